"""Pins for the commit oracle (CPU only).

The commit appends the keys and values of the root and the accepted nodes to
the context cache (the walk of Def. 1 commits them; Eq. 1).  The main pin is
the tiny float64 decoder: GLANCE rounds over a persistent cache, each round
committing its path, must end with the cache that a causal forward over the
committed prefix builds, and with the greedy autoregressive stream (Thm. 1).
A planted mistake (committing nodes 0..a in index order instead of the path)
must break it."""

import numpy as np
import pytest

from oracle import commit as C
from oracle import tiny_model as T
from workloads import trees

N_GEN = 32


@pytest.fixture(scope="module")
def setup():
    for seed in range(20):
        m = T.TinyDecoder(seed)
        prompt = np.random.default_rng(seed + 1000).integers(0, m.vocab, size=6).tolist()
        ar, margins = T.greedy_ar(m, prompt, N_GEN)
        if min(margins) > 1e-6 and len(set(ar)) >= 10:
            return m, prompt, ar
    pytest.fail("no seed with a clear argmax margin")


def _random_proposer(n, seed, vocab):
    state = {"k": 0}

    def propose(ctx, root):
        state["k"] += 1
        par, tok = trees.best_first_tree(n, 6, (1, 2, 3), vocab, (seed, state["k"]))
        tok[0] = root
        return par, tok
    return propose


def _spine_proposer(ar, prompt, vocab, depth, n_side):
    """The true greedy continuation as a spine, side branches hung first so that
    node index and depth disagree."""
    full = list(prompt) + list(ar)
    rng = np.random.default_rng(3)

    def propose(ctx, root):
        pos = len(ctx) + 1
        spine = full[pos:pos + depth]
        parents, tokens = [-1], [int(root)]
        for _ in range(n_side):                       # side children of the root
            t = int(rng.integers(0, vocab))
            if t in tokens[1:] or (spine and t == spine[0]):
                continue
            parents.append(0)
            tokens.append(t)
        prev = 0
        for t in spine:
            parents.append(prev)
            tokens.append(int(t))
            prev = len(parents) - 1
        return np.asarray(parents), np.asarray(tokens)
    return propose


def _check_cache_equals_causal(m, prompt, out, caches, ctx):
    committed = list(prompt) + list(out[:ctx - len(prompt)])
    assert len(committed) == ctx
    _, ref = m.forward_causal(committed)
    for (kc, vc), (k, v) in zip(caches, ref):
        np.testing.assert_allclose(kc[:, :ctx], np.transpose(k, (1, 0, 2)), rtol=0, atol=1e-10)
        np.testing.assert_allclose(vc[:, :ctx], np.transpose(v, (1, 0, 2)), rtol=0, atol=1e-10)


@pytest.mark.parametrize("kind", ["random", "spine", "root_only"])
def test_committed_cache_equals_the_autoregressive_cache(setup, kind):
    m, prompt, ar = setup
    if kind == "random":
        prop = _random_proposer(10, 4, m.vocab)
    elif kind == "spine":
        prop = _spine_proposer(ar, prompt, m.vocab, 4, 3)
    else:
        prop = lambda ctx, root: (np.array([-1]), np.array([root]))
    out, acc, caches, ctx = T.glance_decode_cached(m, prompt, N_GEN, prop)
    assert out == ar
    # each round adds the root and its a accepted tokens (the bonus token is the next root)
    assert ctx == len(prompt) + sum(a + 1 for a in acc)
    _check_cache_equals_causal(m, prompt, out, caches, ctx)
    if kind == "spine":
        assert all(a == 4 for a in acc[:-1])


def test_commit_in_index_order_is_caught(setup, monkeypatch):
    m, prompt, ar = setup
    orig = C.commit_kv

    def index_order(k_ctx, v_ctx, ctx_lens, k_new, v_new, accept_len, accept_path):
        wrong = np.arange(accept_path.shape[1])[None, :].repeat(accept_path.shape[0], 0)
        return orig(k_ctx, v_ctx, ctx_lens, k_new, v_new, accept_len, wrong)
    monkeypatch.setattr(C, "commit_kv", index_order)
    out, acc, caches, ctx = T.glance_decode_cached(m, prompt, N_GEN, _spine_proposer(ar, prompt, m.vocab, 4, 3))
    with pytest.raises(AssertionError):
        assert out == ar
        _check_cache_equals_causal(m, prompt, out, caches, ctx)


def test_hand_worked_commit():
    # batch 2, Hkv 1, D 2, capacity 6; node rows carry their own index
    k_ctx = np.zeros((2, 1, 6, 2))
    v_ctx = np.zeros((2, 1, 6, 2))
    k_new = np.arange(2 * 5, dtype=float).reshape(2, 5, 1, 1).repeat(2, axis=3)
    v_new = -k_new
    path = np.array([[0, 2, 4, -1], [0, -1, -1, -1]])
    kc, vc, lens = C.commit_kv(k_ctx, v_ctx, [1, 4], k_new, v_new, [2, 0], path)
    assert lens.tolist() == [4, 5]
    assert kc[0, 0, :, 0].tolist() == [0, 0, 2, 4, 0, 0]       # slots 1..3 <- nodes 0, 2, 4 of sequence 0
    assert kc[1, 0, :, 0].tolist() == [0, 0, 0, 0, 5, 0]       # slot 4 <- node 0 of sequence 1 (value 5)
    assert vc[0, 0, 2, 1] == -2 and vc[1, 0, 4, 0] == -5
    assert k_ctx.sum() == 0                                     # inputs untouched


def test_capacity_and_invalid_entries():
    k_ctx = np.zeros((1, 2, 4, 3))
    k_new = np.ones((1, 6, 2, 3))
    kc, _, lens = C.commit_kv(k_ctx, k_ctx, [2], k_new, k_new, [3], np.array([[0, 1, 2, 3]]))
    assert lens.tolist() == [4] and kc[0, :, 2:, :].min() == 1  # two slots written, length capped
    kc, _, lens = C.commit_kv(k_ctx, k_ctx, [0], k_new, k_new, [3], np.array([[0, 7, 2, 3]]))
    assert lens.tolist() == [1] and kc[0, :, 1:, :].max() == 0  # entry 7 is not a node: copy stops
    kc, _, lens = C.commit_kv(k_ctx, k_ctx, [0], k_new, k_new, [5], np.array([[0, 1]]))
    assert lens.tolist() == [2]                                 # only path_stride rows exist
