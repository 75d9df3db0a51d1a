"""Explicit-mask float64 attention: the oracle for block-draft and tree-verify.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

What is computed (per sequence b, query head h, new row i):

    keys    = [K_ctx[b, g, 0:ctx_b] ; K_new[b, 0:n, g]]       g = h // (Hq/Hkv)
    values  = [V_ctx[b, g, 0:ctx_b] ; V_new[b, 0:n, g]]
    S[i, j] = sm_scale * <q_i, key_j>,  S[i, j] = -inf where key j is not visible
    O[i]    = sum_j softmax(S[i])_j * value_j,   LSE[i] = log sum_j exp(S[i, j])

Visibility of the context keys: every new row sees every context key (the
context is the cached multimodal prefix x, Sec. 3.1).

Visibility of the new keys:

* block draft (Sec. 3.2): the block is the pending root b followed by B-1 mask
  tokens, drafted in one pass by a block-diffusion head; attention inside the
  block is bidirectional, so every block row sees every block key;
* tree verify (Def. 1, Sec. 3.3; Algorithm 1, App. B): root b and the candidate
  tree are packed behind an ancestor mask, so the row of node i sees node j iff
  j is i itself or an ancestor of i.  That is what makes the row of a depth-d
  node equal to the target distribution after x o b o y_{1:d}.

Readings where the paper is silent: the softmax scale defaults to
1/sqrt(head_dim); query head h reads KV head h // (Hq/Hkv) (contiguous grouped
query attention); the root is new row 0 and is not part of the context.

Every step is a plain numpy float64 operation over an explicit boolean mask;
there is no blocking, no online softmax and no split of the keys.
"""

import math

import numpy as np


def _f64(x):
    """Upcast an array-like (numpy, or a CPU torch tensor of any float dtype) to float64."""
    if hasattr(x, "detach"):  # torch tensor; bf16 upcasts exactly through float32
        x = x.detach().to("cpu")
        if str(x.dtype) in ("torch.bfloat16", "torch.float16"):
            x = x.float()
        x = x.numpy()
    return np.asarray(x, dtype=np.float64)


def _i64(x):
    if hasattr(x, "detach"):
        x = x.detach().to("cpu").numpy()
    return np.asarray(x, dtype=np.int64)


def tree_visibility(parents):
    """Ancestor-or-self visibility of a packed tree (Def. 1; Algorithm 1's ancestor mask).

    ``parents[0] == -1`` is the root b; every other node's parent has a smaller
    index.  Returns a bool matrix vis[i, j] = (j == i or j is an ancestor of i),
    found by walking each node's parent chain up to the root.
    """
    parents = [int(p) for p in _i64(parents)]
    n = len(parents)
    vis = np.zeros((n, n), dtype=bool)
    for i in range(n):
        j = i
        steps = 0
        while j >= 0:
            vis[i, j] = True
            j = parents[j]
            steps += 1
            if steps > n:
                raise ValueError("parents do not form a tree rooted at node 0")
    return vis


def block_visibility(n):
    """Bidirectional block of a block-diffusion draft (Sec. 3.2): every row sees every block key."""
    return np.ones((n, n), dtype=bool)


def masked_attention_one(q, k_ctx, v_ctx, k_new, v_new, ctx_len, visible, sm_scale=None, rows=None):
    """Attention for one sequence.

    q        [n][Hq][D]           new-row queries (post-rotary)
    k_ctx    [Hkv][>=ctx_len][D]  cached context keys; only [:ctx_len] is read
    v_ctx    [Hkv][>=ctx_len][D]
    k_new    [n][Hkv][D]          keys of the new rows (block or packed tree)
    v_new    [n][Hkv][D]
    visible  [n][n] bool          visibility among the new rows
    rows     optional list of new-row indices to evaluate (default: all)

    Returns (out [len(rows)][Hq][D], lse [len(rows)][Hq]) in float64.
    """
    q, k_ctx, v_ctx, k_new, v_new = (_f64(t) for t in (q, k_ctx, v_ctx, k_new, v_new))
    visible = np.asarray(visible, dtype=bool)
    n, hq, d = q.shape
    hkv = k_new.shape[1]
    if hq % hkv:
        raise ValueError("query heads must be a multiple of KV heads")
    group = hq // hkv
    if sm_scale is None or sm_scale <= 0:
        sm_scale = 1.0 / math.sqrt(d)
    ctx_len = int(ctx_len)
    if rows is None:
        rows = list(range(n))
    rows = [int(r) for r in rows]

    out = np.zeros((len(rows), hq, d))
    lse = np.zeros((len(rows), hq))
    # mask over [context keys ; new keys] for the selected rows
    mask = np.concatenate([np.ones((len(rows), ctx_len), dtype=bool), visible[rows, :]], axis=1)
    for h in range(hq):
        g = h // group
        keys = np.concatenate([k_ctx[g, :ctx_len, :], k_new[:, g, :]], axis=0)
        vals = np.concatenate([v_ctx[g, :ctx_len, :], v_new[:, g, :]], axis=0)
        s = sm_scale * (q[rows, h, :] @ keys.T)
        s = np.where(mask, s, -np.inf)
        m = s.max(axis=1, keepdims=True)
        p = np.exp(s - m)
        l = p.sum(axis=1, keepdims=True)
        out[:, h, :] = (p @ vals) / l
        lse[:, h] = (m + np.log(l))[:, 0]
    return out, lse


def block_draft_attn(q, k_ctx, v_ctx, k_new, v_new, ctx_lens, sm_scale=None, rows=None):
    """One-pass block-draft attention (Sec. 3.2), batched.

    q [batch][B][Hq][D]; k_ctx/v_ctx [batch][Hkv][cap][D]; k_new/v_new [batch][B][Hkv][D];
    ctx_lens [batch].  Returns (out [batch][B or len(rows)][Hq][D], lse [batch][..][Hq]).
    """
    ctx_lens = _i64(ctx_lens)
    batch, n = q.shape[0], q.shape[1]
    vis = block_visibility(n)
    outs, lses = [], []
    for b in range(batch):
        o, l = masked_attention_one(q[b], k_ctx[b], v_ctx[b], k_new[b], v_new[b],
                                    ctx_lens[b], vis, sm_scale, rows)
        outs.append(o)
        lses.append(l)
    return np.stack(outs), np.stack(lses)


def tree_verify_attn(q, k_ctx, v_ctx, k_new, v_new, ctx_lens, parents, sm_scale=None, rows=None):
    """One-pass ancestor-masked tree verification (Def. 1; Algorithm 1), batched.

    parents [batch][n] with parents[b][0] = -1 (row 0 is the root b).
    """
    ctx_lens = _i64(ctx_lens)
    parents = _i64(parents)
    batch = q.shape[0]
    outs, lses = [], []
    for b in range(batch):
        vis = tree_visibility(parents[b])
        o, l = masked_attention_one(q[b], k_ctx[b], v_ctx[b], k_new[b], v_new[b],
                                    ctx_lens[b], vis, sm_scale, rows)
        outs.append(o)
        lses.append(l)
    return np.stack(outs), np.stack(lses)
