"""Tiny random-weight float64 decoder for the lossless-greedy check (Thm. 1).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Thm. 1 (Sec. 3.3; full statement and proof in App. A.1): if the target's argmax
is unique at every visited prefix with a margin above the packed-versus-unpacked
perturbation, then for ANY candidate tree the walk of Def. 1 / Algorithm 1
commits exactly the target's greedy autoregressive sequence.

This module builds a small decoder-only transformer with random weights
(RMSNorm, grouped-query attention with rotary positions, SwiGLU MLP, LM head)
and offers two decoders over it:

* ``greedy_ar``      -- plain greedy decoding, one full causal forward per token;
* ``glance_decode``  -- GLANCE rounds (Algorithm 1, App. B): the pending root b and
  a candidate tree are packed into one verify pass whose attention is the
  oracle's explicit-mask attention with the ancestor mask, the node at depth d
  sitting at position ctx + d; the rows are walked by ``oracle.accept``;
* ``glance_decode_cached`` -- the same rounds over a persistent key/value cache:
  the verify pass reads the cache and returns every node's keys and values,
  and the accepted path is committed into the cache by ``oracle.commit``.

The tree proposer is a plug-in argument, standing in for the block head and the
tree builder, which need trained weights.  Whatever it proposes, the committed
stream must equal ``greedy_ar`` token for token.
"""

import numpy as np

from . import attention as _attn
from . import accept as _acc
from . import commit as _commit


class TinyDecoder:
    def __init__(self, seed, vocab=64, d_model=32, n_layers=2, n_q_heads=4, n_kv_heads=2,
                 head_dim=8, d_ff=64, rope_base=10000.0):
        rng = np.random.default_rng(seed)
        self.vocab, self.d_model, self.n_layers = vocab, d_model, n_layers
        self.hq, self.hkv, self.hd, self.d_ff = n_q_heads, n_kv_heads, head_dim, d_ff
        self.rope_base = rope_base
        s = 1.0 / np.sqrt(d_model)
        self.emb = rng.normal(0.0, 1.0, (vocab, d_model))
        self.layers = []
        for _ in range(n_layers):
            self.layers.append({
                "norm1": 1.0 + 0.1 * rng.normal(size=d_model),
                "wq": rng.normal(0.0, s, (d_model, n_q_heads * head_dim)),
                "wk": rng.normal(0.0, s, (d_model, n_kv_heads * head_dim)),
                "wv": rng.normal(0.0, s, (d_model, n_kv_heads * head_dim)),
                "wo": rng.normal(0.0, 1.0 / np.sqrt(n_q_heads * head_dim), (n_q_heads * head_dim, d_model)),
                "norm2": 1.0 + 0.1 * rng.normal(size=d_model),
                "wg": rng.normal(0.0, s, (d_model, d_ff)),
                "wu": rng.normal(0.0, s, (d_model, d_ff)),
                "wd": rng.normal(0.0, 1.0 / np.sqrt(d_ff), (d_ff, d_model)),
            })
        self.norm_f = 1.0 + 0.1 * rng.normal(size=d_model)
        self.lm_head = rng.normal(0.0, 3.0 * s, (d_model, vocab))

    # ---- building blocks -------------------------------------------------
    @staticmethod
    def _rmsnorm(x, g, eps=1e-6):
        return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g

    def _rope(self, x, positions):
        """Rotary embedding, half-split convention; x [T][H][D], positions [T]."""
        d = self.hd
        half = d // 2
        inv = self.rope_base ** (-np.arange(half) * 2.0 / d)
        ang = np.asarray(positions, dtype=np.float64)[:, None] * inv[None, :]
        cos, sin = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
        x1, x2 = x[..., :half], x[..., half:]
        return np.concatenate([x1 * cos - x2 * sin, x1 * sin + x2 * cos], axis=-1)

    def _qkv(self, lw, h, positions):
        t = h.shape[0]
        x = self._rmsnorm(h, lw["norm1"])
        q = (x @ lw["wq"]).reshape(t, self.hq, self.hd)
        k = (x @ lw["wk"]).reshape(t, self.hkv, self.hd)
        v = (x @ lw["wv"]).reshape(t, self.hkv, self.hd)
        return self._rope(q, positions), self._rope(k, positions), v

    def _mlp_residual(self, lw, h, attn_out):
        h = h + attn_out.reshape(h.shape[0], -1) @ lw["wo"]
        x = self._rmsnorm(h, lw["norm2"])
        gate = x @ lw["wg"]
        act = gate / (1.0 + np.exp(-gate)) * (x @ lw["wu"])
        return h + act @ lw["wd"]

    def _logits(self, h):
        return self._rmsnorm(h, self.norm_f) @ self.lm_head

    # ---- plain causal forward (the autoregressive reference) -------------
    def _causal_attention(self, q, k, v):
        """Causal attention written as a loop over query positions."""
        t = q.shape[0]
        g = self.hq // self.hkv
        out = np.zeros_like(q)
        scale = 1.0 / np.sqrt(self.hd)
        for i in range(t):
            for h in range(self.hq):
                s = scale * (k[: i + 1, h // g, :] @ q[i, h, :])
                w = np.exp(s - s.max())
                w /= w.sum()
                out[i, h, :] = w @ v[: i + 1, h // g, :]
        return out

    def forward_causal(self, tokens):
        """Logits [T][vocab] and per-layer (K, V) [T][Hkv][D] of a causal pass over ``tokens``."""
        tokens = np.asarray(tokens, dtype=np.int64)
        pos = np.arange(len(tokens))
        h = self.emb[tokens]
        cache = []
        for lw in self.layers:
            q, k, v = self._qkv(lw, h, pos)
            cache.append((k, v))
            h = self._mlp_residual(lw, h, self._causal_attention(q, k, v))
        return self._logits(h), cache

    # ---- packed tree verify pass (Algorithm 1, "pack b and T") ----------
    def verify_tree(self, ctx_tokens, parents, tokens):
        """Logits [n][vocab] of one ancestor-masked pass over root + tree.

        ctx_tokens are the committed prefix before the root; tokens[0] is the root b.
        Node i sits at position len(ctx) + depth(i).
        """
        ctx_tokens = np.asarray(ctx_tokens, dtype=np.int64)
        tokens = np.asarray(tokens, dtype=np.int64)
        parents = [int(p) for p in parents]
        n = len(parents)
        depth = [0] * n
        for i in range(1, n):
            depth[i] = depth[parents[i]] + 1
        ctx = len(ctx_tokens)
        pos = ctx + np.asarray(depth)
        vis = _attn.tree_visibility(parents)
        if ctx > 0:
            _, cache = self.forward_causal(ctx_tokens)
        h = self.emb[tokens]
        for li, lw in enumerate(self.layers):
            q, k, v = self._qkv(lw, h, pos)
            if ctx > 0:
                kc = np.transpose(cache[li][0], (1, 0, 2))  # [Hkv][ctx][D]
                vc = np.transpose(cache[li][1], (1, 0, 2))
            else:
                kc = np.zeros((self.hkv, 0, self.hd))
                vc = np.zeros((self.hkv, 0, self.hd))
            o, _ = _attn.masked_attention_one(q, kc, vc, k, v, ctx, vis, 1.0 / np.sqrt(self.hd))
            h = self._mlp_residual(lw, h, o)
        return self._logits(h)


    def verify_tree_cached(self, caches, ctx, parents, tokens):
        """The verify pass over a cache: caches[l] = (K, V) [Hkv][capacity][D] holding
        the first ``ctx`` prefix positions.  Returns the rows' logits [n][vocab] and,
        per layer, the nodes' keys and values [n][Hkv][D] (post-rotary, node i at
        position ctx + depth(i))."""
        tokens = np.asarray(tokens, dtype=np.int64)
        parents = [int(p) for p in parents]
        n = len(parents)
        depth = [0] * n
        for i in range(1, n):
            depth[i] = depth[parents[i]] + 1
        pos = ctx + np.asarray(depth)
        vis = _attn.tree_visibility(parents)
        h = self.emb[tokens]
        new_kv = []
        for li, lw in enumerate(self.layers):
            q, k, v = self._qkv(lw, h, pos)
            new_kv.append((k, v))
            kc, vc = caches[li][0][:, :ctx], caches[li][1][:, :ctx]
            o, _ = _attn.masked_attention_one(q, kc, vc, k, v, ctx, vis, 1.0 / np.sqrt(self.hd))
            h = self._mlp_residual(lw, h, o)
        return self._logits(h), new_kv


def greedy_ar(model, prompt, n_tokens):
    """Greedy autoregressive decoding (Sec. 3.1): one full forward per token.

    Returns (tokens, margins): the n_tokens generated ids and the top-2 logit gap at each step.
    """
    seq = list(int(t) for t in prompt)
    out, margins = [], []
    for _ in range(n_tokens):
        logits, _ = model.forward_causal(seq)
        row = logits[-1]
        top = np.sort(row)[-2:]
        margins.append(float(top[1] - top[0]))
        t = int(np.argmax(row))
        out.append(t)
        seq.append(t)
    return out, margins


def glance_decode(model, prompt, n_tokens, propose_tree):
    """GLANCE rounds (Algorithm 1, App. B) with a plug-in tree proposer.

    propose_tree(ctx_tokens, root) -> (parents, tokens) with tokens[0] == root.
    Returns (generated tokens, list of accepted lengths a per round).
    """
    prompt = [int(t) for t in prompt]
    logits, _ = model.forward_causal(prompt)
    out = [int(np.argmax(logits[-1]))]  # the first pending root comes from the prefill
    accepted = []
    while len(out) < n_tokens:
        ctx = prompt + out[:-1]
        root = out[-1]
        parents, tokens = propose_tree(ctx, root)
        if int(tokens[0]) != root or int(parents[0]) != -1:
            raise ValueError("tree row 0 must be the pending root")
        rows = model.verify_tree(ctx, parents, tokens)
        am = _acc.argmax_rows(rows)
        a, path, nr = _acc.greedy_walk(am, parents, tokens)
        accepted.append(a)
        out.extend(int(tokens[c]) for c in path[1:])
        out.append(int(nr))
    return out[:n_tokens], accepted


def glance_decode_cached(model, prompt, n_tokens, propose_tree, capacity=256):
    """GLANCE rounds over a persistent cache, committing each round's path.

    Returns (generated tokens, accepted lengths, caches, ctx): caches[l] = (K, V)
    [Hkv][capacity][D] after the last round and ctx the committed prefix length
    (prompt + every committed token except the pending root).
    """
    prompt = [int(t) for t in prompt]
    logits, pre = model.forward_causal(prompt)
    caches = []
    for k, v in pre:
        kc = np.zeros((model.hkv, capacity, model.hd))
        vc = np.zeros((model.hkv, capacity, model.hd))
        kc[:, :len(prompt)] = np.transpose(k, (1, 0, 2))
        vc[:, :len(prompt)] = np.transpose(v, (1, 0, 2))
        caches.append((kc, vc))
    ctx = len(prompt)
    out = [int(np.argmax(logits[-1]))]
    accepted = []
    while len(out) < n_tokens:
        root = out[-1]
        parents, tokens = propose_tree(prompt + out[:-1], root)
        rows, new_kv = model.verify_tree_cached(caches, ctx, parents, tokens)
        am = _acc.argmax_rows(rows)
        a, path, nr = _acc.greedy_walk(am, parents, tokens)
        accepted.append(a)
        path_arr = np.asarray([path], dtype=np.int64)
        for li in range(len(caches)):
            k_new, v_new = new_kv[li]
            kc, vc, lens = _commit.commit_kv(caches[li][0][None], caches[li][1][None], [ctx],
                                             k_new[None], v_new[None], [a], path_arr)
            caches[li] = (kc[0], vc[0])
        ctx = int(lens[0])
        out.extend(int(tokens[c]) for c in path[1:])
        out.append(int(nr))
    return out[:n_tokens], accepted, caches, ctx
