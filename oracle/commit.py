"""Commit oracle: the accepted path's keys and values join the context cache.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

After the walk (Def. 1, Algorithm 1) a round commits the pending root b and
the accepted tokens y_1..y_a: these a + 1 tokens join the prefix, and the
bonus token becomes the next root (Sec. 3.1, Eq. 1).  The verify pass has
already computed the target's keys and values of every tree node, each node
at position ctx + depth, which for the nodes of the accepted path is exactly
the cache slot the token occupies in the prefix.  Committing is therefore a
gather: cache slot ctx + i receives the row of path node i (i = 0..a), and the
context length grows by a + 1.  ``tests/test_oracle_commit.py`` pins this
against autoregressive decoding of the tiny model: the cache built round by
round equals the one a causal forward over the committed prefix builds.

Layouts (as on the GPU path):
  k_ctx, v_ctx  [batch][Hkv][capacity][D]     k_new, v_new  [batch][n][Hkv][D]
  ctx_lens      [batch]                       accept_len [batch], accept_path [batch][stride]
"""

import numpy as np


def commit_kv(k_ctx, v_ctx, ctx_lens, k_new, v_new, accept_len, accept_path):
    """Returns (k_ctx', v_ctx', ctx_lens') after committing every sequence's path.

    Slots at or past the capacity are not written and the length stops at the
    capacity; a path entry outside [0, n) ends that sequence's copy (the
    length then grows by the rows copied).  Inputs are not modified.
    """
    k_ctx = np.array(k_ctx, copy=True)
    v_ctx = np.array(v_ctx, copy=True)
    lens = np.array(ctx_lens, dtype=np.int64, copy=True)
    batch, n = k_new.shape[0], k_new.shape[1]
    cap = k_ctx.shape[2]
    stride = accept_path.shape[1]
    for b in range(batch):
        ctx = int(lens[b])
        rows = min(int(accept_len[b]) + 1, stride, n)
        copied = 0
        for i in range(rows):
            node = int(accept_path[b][i])
            if node < 0 or node >= n:
                break
            if ctx + i < cap:
                k_ctx[b, :, ctx + i, :] = k_new[b, node]
                v_ctx[b, :, ctx + i, :] = v_new[b, node]
            copied += 1
        lens[b] = min(ctx + copied, cap)
    return k_ctx, v_ctx, lens
