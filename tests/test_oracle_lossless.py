"""Thm. 1 on a tiny random-weight float64 decoder (CPU only).

Whatever tree is proposed, GLANCE rounds must commit exactly the greedy
autoregressive stream.  The "perfect" proposer, which contains the true
continuation, additionally checks that a depth-d row of the packed pass really
is the target distribution after x o b o y_{1:d} (Def. 1): otherwise its
accepted lengths would fall short of the tree depth.

Two planted mistakes in the oracle (on the CPU) show the check has teeth: a
causal-by-index mask instead of the ancestor mask, and positions ctx + index
instead of ctx + depth, both break losslessness on branching trees.
"""

import numpy as np
import pytest

from oracle import attention as A
from oracle import tiny_model as T
from workloads import trees

N_GEN = 40


def _model_and_ar(seed):
    m = T.TinyDecoder(seed)
    prompt = np.random.default_rng(seed + 1000).integers(0, m.vocab, size=6).tolist()
    ar, margins = T.greedy_ar(m, prompt, N_GEN)
    return m, prompt, ar, margins


@pytest.fixture(scope="module")
def setup():
    for seed in range(20):
        m, prompt, ar, margins = _model_and_ar(seed)
        # the theorem's unique-argmax assumption with room to spare, and a non-degenerate stream
        if min(margins) > 1e-6 and len(set(ar)) >= 12:
            return m, prompt, ar
    pytest.fail("no seed with a clear argmax margin")


def _renumber_topologically(parents, tokens, rng):
    """Renumber a tree in a random topological order (parents keep smaller indices, root stays 0)."""
    n = len(parents)
    order, placed = [0], {0}
    while len(order) < n:
        ready = [c for c in range(n) if c not in placed and parents[c] in placed]
        c = ready[int(rng.integers(0, len(ready)))]
        order.append(c)
        placed.add(c)
    new_of = {old: new for new, old in enumerate(order)}
    par = [-1 if parents[o] < 0 else new_of[parents[o]] for o in order]
    tok = [tokens[o] for o in order]
    return par, tok


def _random_proposer(n, seed, vocab):
    state = {"k": 0}

    def propose(ctx, root):
        state["k"] += 1
        par, tok = trees.best_first_tree(n, 6, (1, 2, 3), vocab, (seed, state["k"]))
        tok[0] = root
        return par, tok
    return propose


def _perfect_proposer(ar, prompt, n_side, vocab, depth):
    """A tree whose spine is the true greedy continuation (depth ``depth``) plus random side branches."""
    full = list(prompt) + list(ar)
    rng = np.random.default_rng(5)

    def propose(ctx, root):
        pos = len(ctx) + 1   # index in ``full`` of the token after the root
        spine = full[pos:pos + depth]
        parents, tokens = [-1], [root]
        for t in spine:
            parents.append(len(parents) - 1)
            tokens.append(t)
        for _ in range(n_side):
            p = int(rng.integers(0, len(parents)))
            used = {tokens[c] for c in range(1, len(parents)) if parents[c] == p}
            t = int(rng.integers(0, vocab))
            if t in used:
                continue
            parents.append(p)
            tokens.append(t)
        # interleave side nodes with the spine so that node index and depth disagree
        return _renumber_topologically(parents, tokens, rng)
    return propose


def test_random_trees_are_lossless(setup):
    m, prompt, ar = setup
    out, acc = T.glance_decode(m, prompt, N_GEN, _random_proposer(12, 1, m.vocab))
    assert out == ar


def test_chain_star_and_root_only_are_lossless(setup):
    m, prompt, ar = setup
    for make in (lambda k: trees.chain_tree(8, m.vocab, (2, k)),
                 lambda k: trees.star_tree(8, m.vocab, (3, k)),
                 lambda k: (np.array([-1]), np.array([0]))):
        cnt = {"k": 0}

        def propose(ctx, root, make=make, cnt=cnt):
            cnt["k"] += 1
            p, t = make(cnt["k"])
            t = np.array(t).copy()
            t[0] = root
            return p, t
        out, acc = T.glance_decode(m, prompt, N_GEN, propose)
        assert out == ar


def test_perfect_tree_accepts_its_full_spine(setup):
    m, prompt, ar = setup
    depth = 5
    out, acc = T.glance_decode(m, prompt, N_GEN, _perfect_proposer(ar, prompt, 6, m.vocab, depth))
    assert out == ar
    # every round but possibly the last (which runs out of reference tokens) accepts the whole spine
    assert all(a == depth for a in acc[:-1])


def test_planted_mask_mistake_is_caught(setup, monkeypatch):
    m, prompt, ar = setup
    monkeypatch.setattr(A, "tree_visibility",
                        lambda parents: np.tril(np.ones((len(parents), len(parents)), dtype=bool)))
    out, acc = T.glance_decode(m, prompt, N_GEN, _perfect_proposer(ar, prompt, 6, m.vocab, 5))
    assert out != ar or any(a < 5 for a in acc[:-1])


def test_planted_position_mistake_is_caught(setup, monkeypatch):
    m, prompt, ar = setup
    orig = T.TinyDecoder.verify_tree

    def by_index(self, ctx_tokens, parents, tokens):
        # positions ctx + index instead of ctx + depth: rebuild as if every node were a chain node
        saved = self._rope

        def rope(x, positions):
            return saved(x, len(ctx_tokens) + np.arange(len(positions)))
        self._rope = rope
        try:
            return orig(self, ctx_tokens, parents, tokens)
        finally:
            del self._rope
    monkeypatch.setattr(T.TinyDecoder, "verify_tree", by_index)

    def side_first(ctx, root):
        # the true spine hangs below a side node, so index != depth on the spine
        full = list(prompt) + list(ar)
        pos = len(ctx) + 1
        parents, tokens = [-1, 0, 0, 0], [root, (full[pos] + 1) % m.vocab, (full[pos] + 2) % m.vocab,
                                          full[pos]]
        for t in full[pos + 1:pos + 4]:
            parents.append(len(parents) - 1)
            tokens.append(t)
        return parents, tokens
    out, acc = T.glance_decode(m, prompt, N_GEN, side_first)
    assert out != ar or any(a < 4 for a in acc[:-1])
