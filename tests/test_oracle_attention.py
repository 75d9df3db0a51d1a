"""Pins for the float64 attention oracle (CPU only).

Each check ties the oracle to something other than itself: hand-derived
closed forms (uniform attention over a hand-listed ancestor set, a two-key
softmax with weights 3/4 and 1/4), library attention (torch SDPA in float64
with a mask built by a different algorithm), and the symmetries the masks
must have (a bidirectional block is permutation-equivariant, a tree is
invariant to relabelling its nodes in another topological order).
"""

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import attention as A

# Hand-listed tree: parents and the ancestor-or-self sets written out by hand (Def. 1).
TREE_PARENTS = [-1, 0, 0, 1, 1, 2, 4, 6, 3]
TREE_ANCESTORS = [
    {0}, {0, 1}, {0, 2}, {0, 1, 3}, {0, 1, 4}, {0, 2, 5}, {0, 1, 4, 6}, {0, 1, 4, 6, 7}, {0, 1, 3, 8},
]


def _rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).normal(0.0, scale, shape)


def test_tree_visibility_matches_hand_listed_ancestors():
    vis = A.tree_visibility(TREE_PARENTS)
    for i, anc in enumerate(TREE_ANCESTORS):
        assert set(np.nonzero(vis[i])[0].tolist()) == anc


@pytest.mark.parametrize("ctx", [0, 5])
def test_uniform_scores_reveal_the_tree_mask(ctx):
    """Q = 0 makes every visible key equally weighted, so with one-hot values the
    output of node i is 1/(ctx + |anc(i)|) on exactly its ancestor columns, and
    LSE = log(ctx + |anc(i)|)."""
    n, hq, hkv, d = len(TREE_PARENTS), 2, 1, 16
    q = np.zeros((1, n, hq, d))
    k_new = _rand((1, n, hkv, d), 1)
    v_new = np.zeros((1, n, hkv, d))
    for j in range(n):
        v_new[0, j, 0, j] = 1.0
    k_ctx = _rand((1, hkv, max(ctx, 1), d), 2)
    v_ctx = np.zeros((1, hkv, max(ctx, 1), d))
    v_ctx[0, 0, :, d - 1] = 1.0  # context mass lands in the last column
    out, lse = A.tree_verify_attn(q, k_ctx, v_ctx, k_new, v_new, [ctx], [TREE_PARENTS])
    for i, anc in enumerate(TREE_ANCESTORS):
        cnt = ctx + len(anc)
        for h in range(hq):
            expect = np.zeros(d)
            for j in anc:
                expect[j] = 1.0 / cnt
            expect[d - 1] += ctx / cnt
            np.testing.assert_allclose(out[0, i, h], expect, atol=1e-15)
            assert lse[0, i, h] == pytest.approx(math.log(cnt), abs=1e-14)


def test_uniform_scores_block_sees_everything():
    n, hq, hkv, d, ctx = 6, 4, 2, 8, 7
    q = np.zeros((1, n, hq, d))
    k_ctx, k_new = _rand((1, hkv, ctx, d), 3), _rand((1, n, hkv, d), 4)
    v_ctx, v_new = _rand((1, hkv, ctx, d), 5), _rand((1, n, hkv, d), 6)
    out, lse = A.block_draft_attn(q, k_ctx, v_ctx, k_new, v_new, [ctx])
    for h in range(hq):
        g = h // 2
        mean = (v_ctx[0, g].sum(0) + v_new[0, :, g].sum(0)) / (ctx + n)
        for i in range(n):
            np.testing.assert_allclose(out[0, i, h], mean, atol=1e-15)
            assert lse[0, i, h] == pytest.approx(math.log(ctx + n), abs=1e-14)


def test_two_key_softmax_weights_three_to_one_and_default_scale():
    """Block of one row over one context key: with default scale 1/sqrt(64) = 1/8,
    q = (8 ln 3) e0 and k_ctx = e0, k_new = 0 give scores ln 3 and 0, so the
    softmax weights are exactly 3/4 and 1/4 and LSE = ln 4."""
    d = 64
    q = np.zeros((1, 1, 1, d))
    q[0, 0, 0, 0] = 8.0 * math.log(3.0)
    k_ctx = np.zeros((1, 1, 1, d))
    k_ctx[0, 0, 0, 0] = 1.0
    k_new = np.zeros((1, 1, 1, d))
    v_ctx = np.zeros((1, 1, 1, d))
    v_ctx[0, 0, 0, 0] = 2.0
    v_new = np.zeros((1, 1, 1, d))
    v_new[0, 0, 0, 1] = -4.0
    out, lse = A.block_draft_attn(q, k_ctx, v_ctx, k_new, v_new, [1])
    expect = np.zeros(d)
    expect[0] = 0.75 * 2.0
    expect[1] = 0.25 * -4.0
    np.testing.assert_allclose(out[0, 0, 0], expect, atol=1e-14)
    assert lse[0, 0, 0] == pytest.approx(math.log(4.0), abs=1e-14)


def test_gqa_contiguous_grouping():
    """Query head h reads KV head h // (Hq/Hkv): KV head g carries constant value g+1."""
    n, hq, hkv, d, ctx = 3, 6, 3, 8, 4
    q = _rand((1, n, hq, d), 7)
    k_ctx, k_new = _rand((1, hkv, ctx, d), 8), _rand((1, n, hkv, d), 9)
    v_ctx = np.zeros((1, hkv, ctx, d))
    v_new = np.zeros((1, n, hkv, d))
    for g in range(hkv):
        v_ctx[0, g] = g + 1.0
        v_new[0, :, g] = g + 1.0
    out, _ = A.block_draft_attn(q, k_ctx, v_ctx, k_new, v_new, [ctx])
    for h in range(hq):
        np.testing.assert_allclose(out[0, :, h], h // 2 + 1.0, atol=1e-14)


def _sdpa(q_rows, keys, vals, mask, scale):
    """torch SDPA in float64: q_rows [R][D], keys/vals [K][D], mask [R][K] bool."""
    o = F.scaled_dot_product_attention(
        torch.from_numpy(q_rows)[None, None], torch.from_numpy(keys)[None, None],
        torch.from_numpy(vals)[None, None], attn_mask=torch.from_numpy(mask)[None, None],
        scale=scale)
    return o[0, 0].numpy()


def _closure_mask(parents):
    """Ancestor-or-self by transitive closure of the child->parent adjacency (boolean matrix powers)."""
    n = len(parents)
    adj = np.zeros((n, n), dtype=np.int64)
    for c, p in enumerate(parents):
        if p >= 0:
            adj[c, p] = 1
    reach = np.eye(n, dtype=np.int64)
    step = np.eye(n, dtype=np.int64)
    for _ in range(n):
        step = (step @ adj > 0).astype(np.int64)
        reach = ((reach + step) > 0).astype(np.int64)
    return reach.astype(bool)


@pytest.mark.parametrize("shape", ["random", "chain", "star"])
def test_verify_matches_sdpa_with_independently_built_mask(shape):
    rng = np.random.default_rng(11)
    n, hq, hkv, d, ctx = 12, 4, 2, 16, 9
    if shape == "chain":
        parents = list(range(-1, n - 1))
    elif shape == "star":
        parents = [-1] + [0] * (n - 1)
    else:
        parents = [-1] + [int(rng.integers(0, i)) for i in range(1, n)]
    q = _rand((1, n, hq, d), 12)
    k_ctx, v_ctx = _rand((1, hkv, ctx + 3, d), 13), _rand((1, hkv, ctx + 3, d), 14)
    k_new, v_new = _rand((1, n, hkv, d), 15), _rand((1, n, hkv, d), 16)
    scale = 0.37
    out, lse = A.tree_verify_attn(q, k_ctx, v_ctx, k_new, v_new, [ctx], [parents], sm_scale=scale)
    tail = _closure_mask(parents)
    if shape == "chain":  # a chain must be plain causal attention over ctx + chain
        np.testing.assert_array_equal(tail, np.tril(np.ones((n, n), dtype=bool)))
    if shape == "star":   # a star node sees the context, the root and itself
        expect = np.zeros((n, n), dtype=bool)
        expect[:, 0] = True
        expect[np.arange(n), np.arange(n)] = True
        np.testing.assert_array_equal(tail, expect)
    mask = np.concatenate([np.ones((n, ctx), dtype=bool), tail], axis=1)
    for h in range(hq):
        g = h // 2
        keys = np.concatenate([k_ctx[0, g, :ctx], k_new[0, :, g]])
        vals = np.concatenate([v_ctx[0, g, :ctx], v_new[0, :, g]])
        ref = _sdpa(q[0, :, h], keys, vals, mask, scale)
        np.testing.assert_allclose(out[0, :, h], ref, atol=1e-12)
        s = scale * q[0, :, h] @ keys.T
        s[~mask] = -np.inf
        ref_lse = torch.logsumexp(torch.from_numpy(s), dim=1).numpy()
        np.testing.assert_allclose(lse[0, :, h], ref_lse, atol=1e-12)


def test_block_length_one_is_plain_decode_attention():
    hq, hkv, d, ctx = 4, 1, 32, 20
    q = _rand((1, 1, hq, d), 20)
    k_ctx, v_ctx = _rand((1, hkv, ctx, d), 21), _rand((1, hkv, ctx, d), 22)
    k_new, v_new = _rand((1, 1, hkv, d), 23), _rand((1, 1, hkv, d), 24)
    for fn in (lambda: A.block_draft_attn(q, k_ctx, v_ctx, k_new, v_new, [ctx]),
               lambda: A.tree_verify_attn(q, k_ctx, v_ctx, k_new, v_new, [ctx], [[-1]])):
        out, _ = fn()
        for h in range(hq):
            keys = np.concatenate([k_ctx[0, 0], k_new[0, :, 0]])
            vals = np.concatenate([v_ctx[0, 0], v_new[0, :, 0]])
            o = F.scaled_dot_product_attention(
                torch.from_numpy(q[0, :, h])[None, None], torch.from_numpy(keys)[None, None],
                torch.from_numpy(vals)[None, None])[0, 0].numpy()
            np.testing.assert_allclose(out[0, :, h], o, atol=1e-12)


def test_block_draft_is_permutation_equivariant():
    """A bidirectional block: permuting block rows together with block keys permutes the output.
    A causal block would fail this."""
    n, hq, hkv, d, ctx = 7, 4, 2, 16, 5
    q = _rand((1, n, hq, d), 30, 2.0)
    k_ctx, v_ctx = _rand((1, hkv, ctx, d), 31), _rand((1, hkv, ctx, d), 32)
    k_new, v_new = _rand((1, n, hkv, d), 33, 2.0), _rand((1, n, hkv, d), 34)
    out, lse = A.block_draft_attn(q, k_ctx, v_ctx, k_new, v_new, [ctx])
    perm = np.random.default_rng(35).permutation(n)
    out2, lse2 = A.block_draft_attn(q[:, perm], k_ctx, v_ctx, k_new[:, perm], v_new[:, perm], [ctx])
    np.testing.assert_allclose(out2, out[:, perm], atol=1e-12)
    np.testing.assert_allclose(lse2, lse[:, perm], atol=1e-12)


def test_tree_relabelling_permutes_outputs():
    """Renumbering the nodes in another topological order (parents still < child) permutes rows."""
    parents = TREE_PARENTS
    n, hq, hkv, d, ctx = len(parents), 4, 2, 8, 6
    q = _rand((1, n, hq, d), 40, 2.0)
    k_ctx, v_ctx = _rand((1, hkv, ctx, d), 41), _rand((1, hkv, ctx, d), 42)
    k_new, v_new = _rand((1, n, hkv, d), 43, 2.0), _rand((1, n, hkv, d), 44)
    out, lse = A.tree_verify_attn(q, k_ctx, v_ctx, k_new, v_new, [ctx], [parents])
    # another topological order: breadth-first by depth, reversed within a depth
    depth = [0] * n
    for i in range(1, n):
        depth[i] = depth[parents[i]] + 1
    order = sorted(range(n), key=lambda i: (depth[i], -i))  # new index -> old index
    new_of = {old: new for new, old in enumerate(order)}
    par2 = [-1 if parents[old] < 0 else new_of[parents[old]] for old in order]
    assert all(par2[i] < i for i in range(1, n))
    out2, lse2 = A.tree_verify_attn(q[:, order], k_ctx, v_ctx, k_new[:, order], v_new[:, order],
                                    [ctx], [par2])
    np.testing.assert_allclose(out2, out[:, order], atol=1e-12)
    np.testing.assert_allclose(lse2, lse[:, order], atol=1e-12)


def test_hard_attention_limit_selects_the_best_visible_key():
    """With one visible key scoring far above the rest the output is that key's value;
    an invisible key with an even larger score must be ignored (mask applied before softmax)."""
    parents = [-1, 0, 0]
    n, hq, hkv, d, ctx = 3, 1, 1, 8, 4
    q = np.zeros((1, n, hq, d))
    q[0, :, 0, 0] = 1.0
    k_ctx = np.zeros((1, hkv, ctx, d))
    k_new = np.zeros((1, n, hkv, d))
    k_new[0, 0, 0, 0] = 500.0   # root: visible to all nodes
    k_new[0, 1, 0, 0] = 900.0   # node 1: visible only to itself
    v_ctx = _rand((1, hkv, ctx, d), 50)
    v_new = _rand((1, n, hkv, d), 51)
    out, _ = A.tree_verify_attn(q, k_ctx, v_ctx, k_new, v_new, [ctx], [parents], sm_scale=1.0)
    np.testing.assert_allclose(out[0, 0, 0], v_new[0, 0, 0], atol=1e-12)
    np.testing.assert_allclose(out[0, 1, 0], v_new[0, 1, 0], atol=1e-12)
    np.testing.assert_allclose(out[0, 2, 0], v_new[0, 0, 0], atol=1e-12)


def test_row_subset_matches_full_evaluation():
    n, hq, hkv, d, ctx = 10, 4, 2, 16, 12
    parents = [-1, 0, 1, 1, 0, 4, 5, 2, 7, 3]
    q = _rand((2, n, hq, d), 60)
    k_ctx, v_ctx = _rand((2, hkv, ctx, d), 61), _rand((2, hkv, ctx, d), 62)
    k_new, v_new = _rand((2, n, hkv, d), 63), _rand((2, n, hkv, d), 64)
    out, lse = A.tree_verify_attn(q, k_ctx, v_ctx, k_new, v_new, [ctx, 5], [parents, parents])
    rows = [9, 0, 4]
    out_s, lse_s = A.tree_verify_attn(q, k_ctx, v_ctx, k_new, v_new, [ctx, 5], [parents, parents],
                                      rows=rows)
    np.testing.assert_allclose(out_s, out[:, rows], atol=0)
    np.testing.assert_allclose(lse_s, lse[:, rows], atol=0)


def test_bf16_inputs_upcast_exactly():
    t = torch.randn(3, 5).to(torch.bfloat16)
    np.testing.assert_array_equal(A._f64(t), t.float().numpy().astype(np.float64))
