"""Seeded synthetic inputs shaped like the paper's grounded-document workloads.

Inputs only: this module draws random tensors and trees and computes no step
of the method.  Both the oracle and the HIP path consume exactly what it
returns (CPU torch tensors; bf16 values are cast once here with
round-to-nearest-even, so both sides see the same numbers).

The paper decodes with Qwen3-VL-8B at batch 1 over document, chart and
infographic prompts whose images enter the target as a token prefix fused into
the same key-value cache as the text (Sec. 5.1, App. C).  Those datasets and
weights are not available, so these generators stand in for them with the
attention shapes of a Qwen2.5-VL-7B-class target (28 query heads, 4 KV heads,
head_dim 128, bf16 cache), image-prefix-dominated contexts, a 16-token draft
block (B = 16, Sec. 3.2) and a 64-row tree (root + budget 63, Sec. 3.3).

Named workloads:

  tiny_fp32     batch 1, 4/1 heads, D 64, ctx 256 (64 image), fp32, block 8,
                16-row tree (depth <= 6, branching {1,2}), logits 16 x 1000
  draft_2k      batch 1, 28/4/128 bf16, ctx 2048 (1296 image + 752 text), block 16
  verify_4k     batch 1, 28/4/128 bf16, ctx 4096, 64-row tree (depth <= 15,
                branching {1,2,4}), logits 64 x 152064 bf16 ~ N(0, 2)
  doc_16k       batch 4, ctx 16384 (14336 image + 2048 text): block 16, then the
                verify_4k tree/logit generator per sequence: a full round
  ragged_mix    batch 16, ctx ~ U{2048..32768} per sequence (60-90% image),
                per-sequence block 16, tree and logits: a full round

Q, K, V ~ N(0, 1) / sqrt(D) unless a variant overrides it.  Logits get a planted
argmax: for a row whose node has children, with probability p(depth) one child
c is chosen uniformly and logit[tokens[c]] is set to the row maximum + 1, so
the target's greedy token is that child's token.
"""

import dataclasses
import math

import numpy as np
import torch

from . import trees

VOCAB_QWEN = 152064


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    cfg_id: int
    batch: int
    hq: int
    hkv: int
    d: int
    dtype: str              # "f32" or "bf16"
    ctx: int                # fixed context length (ignored if ctx_range is set)
    image: int              # image-token prefix length (metadata)
    n_draft: int
    n_tree: int
    depth_cap: int
    branch: tuple
    vocab: int
    logit_sigma: float
    plant_hi: float
    plant_lo: float
    ctx_range: tuple = None  # (lo, hi) inclusive, per-sequence uniform
    image_frac: tuple = None  # (lo, hi) for ragged_mix metadata
    steps: tuple = ("draft", "verify", "accept")

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    @property
    def cap(self):
        return self.ctx_range[1] if self.ctx_range else self.ctx


WORKLOADS = {
    "tiny_fp32": Workload("tiny_fp32", 0, 1, 4, 1, 64, "f32", 256, 64, 8, 16, 6, (1, 2), 1000,
                          1.0, 0.7, 0.7),
    "draft_2k": Workload("draft_2k", 1, 1, 28, 4, 128, "bf16", 2048, 1296, 16, 64, 15, (1, 2, 4),
                         VOCAB_QWEN, math.sqrt(2.0), 0.9, 0.5, steps=("draft",)),
    "verify_4k": Workload("verify_4k", 2, 1, 28, 4, 128, "bf16", 4096, 3072, 16, 64, 15, (1, 2, 4),
                          VOCAB_QWEN, math.sqrt(2.0), 0.9, 0.5, steps=("verify", "accept")),
    "doc_16k": Workload("doc_16k", 3, 4, 28, 4, 128, "bf16", 16384, 14336, 16, 64, 15, (1, 2, 4),
                        VOCAB_QWEN, math.sqrt(2.0), 0.9, 0.5),
    "ragged_mix": Workload("ragged_mix", 4, 16, 28, 4, 128, "bf16", 0, 0, 16, 64, 15, (1, 2, 4),
                           VOCAB_QWEN, math.sqrt(2.0), 0.9, 0.5, ctx_range=(2048, 32768),
                           image_frac=(0.6, 0.9)),
}


def _seed(*key):
    return int(np.random.SeedSequence([int(k) for k in key]).generate_state(1, np.uint64)[0] >> 1)


def _randn(shape, key, sigma):
    g = torch.Generator().manual_seed(_seed(*key))
    return torch.randn(shape, generator=g, dtype=torch.float32) * sigma


# tensor ids for seeding
_T_Q, _T_KC, _T_VC, _T_KN, _T_VN, _T_LOG, _T_TREE, _T_CTX, _T_PLANT = range(9)
_STEP_DRAFT, _STEP_VERIFY = 0, 1


def context_lengths(w, seed=0):
    if w.ctx_range is None:
        return np.full(w.batch, w.ctx, dtype=np.int32)
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([w.cfg_id, _T_CTX, seed])))
    return rng.integers(w.ctx_range[0], w.ctx_range[1] + 1, size=w.batch).astype(np.int32)


def image_lengths(w, ctx_lens, seed=0):
    """Image-prefix length per sequence (metadata only: image tokens share the cache)."""
    if w.image_frac is None:
        return np.full(w.batch, w.image, dtype=np.int32)
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([w.cfg_id, _T_CTX, seed, 1])))
    frac = rng.uniform(w.image_frac[0], w.image_frac[1], size=w.batch)
    return np.floor(frac * ctx_lens).astype(np.int32)


def attention_inputs(w, step, n_new, ctx_lens, seed=0, variant=None, poison=False, cap=None):
    """Q / context K,V / new K,V for one attention call.

    step      "draft" or "verify" (separate caches: the draft head's and the target's)
    variant   None (config scaling), "sharp1" (Q,K,V ~ N(0,1)), "sharp4" (Q ~ N(0,16)),
              "tree_dominant" (new keys aligned with the queries of their rows)
    poison    fill cache padding beyond ctx_len with NaN (catches unguarded loads)
    """
    sid = _STEP_DRAFT if step == "draft" else _STEP_VERIFY
    ctx_lens = np.asarray(ctx_lens, dtype=np.int64)
    if cap is None:
        cap = int(ctx_lens.max())
    cap = max(int(cap), int(ctx_lens.max()), 1)
    b_, hq, hkv, d = len(ctx_lens), w.hq, w.hkv, w.d
    sq = sk = sv = 1.0 / math.sqrt(d)
    if variant in ("sharp1", "sharp4", "tree_dominant"):
        sq = sk = sv = 1.0
        if variant == "sharp4":
            sq = 4.0
    dt = w.torch_dtype
    q = torch.empty((b_, n_new, hq, d), dtype=dt)
    k_new = torch.empty((b_, n_new, hkv, d), dtype=dt)
    v_new = torch.empty((b_, n_new, hkv, d), dtype=dt)
    fill = float("nan") if poison else 0.0
    k_ctx = torch.full((b_, hkv, cap, d), fill, dtype=dt)
    v_ctx = torch.full((b_, hkv, cap, d), fill, dtype=dt)
    for b in range(b_):
        c = int(ctx_lens[b])
        key = (w.cfg_id, sid, seed, b)
        q[b] = _randn((n_new, hq, d), key + (_T_Q,), sq).to(dt)
        kn = _randn((n_new, hkv, d), key + (_T_KN,), sk)
        if variant == "tree_dominant":
            g = hq // hkv
            qf = q[b].float().reshape(n_new, hkv, g, d).mean(dim=2)
            kn = 3.0 * qf + 0.1 * kn
        k_new[b] = kn.to(dt)
        v_new[b] = _randn((n_new, hkv, d), key + (_T_VN,), sv).to(dt)
        if c > 0:
            k_ctx[b, :, :c] = _randn((hkv, c, d), key + (_T_KC,), sk).to(dt)
            v_ctx[b, :, :c] = _randn((hkv, c, d), key + (_T_VC,), sv).to(dt)
    return {"q": q, "k_ctx": k_ctx, "v_ctx": v_ctx, "k_new": k_new, "v_new": v_new,
            "ctx_lens": torch.as_tensor(np.asarray(ctx_lens, dtype=np.int32))}


def tree_inputs(w, seed=0, shape="best_first", n=None, batch=None):
    """parents / tokens [batch][n] int32 per sequence (shape: best_first, chain or star)."""
    n = n if n is not None else w.n_tree
    batch = batch if batch is not None else w.batch
    par = np.zeros((batch, n), dtype=np.int32)
    tok = np.zeros((batch, n), dtype=np.int32)
    for b in range(batch):
        key = (w.cfg_id, _T_TREE, seed, b)
        if shape == "best_first":
            p, t = trees.best_first_tree(n, w.depth_cap, w.branch, w.vocab, key)
        elif shape == "chain":
            p, t = trees.chain_tree(n, w.vocab, key)
        elif shape == "star":
            p, t = trees.star_tree(n, w.vocab, key)
        else:
            raise ValueError(shape)
        par[b], tok[b] = p, t
    return torch.as_tensor(par), torch.as_tensor(tok)


def planted_logits(w, parents, tokens, seed=0, plant=True):
    """Verified rows [batch][n][V] ~ N(0, sigma^2), with the greedy token planted on a child.

    For each row v that has children: with probability p(depth_v) pick a child c
    uniformly and set logit[tokens[c]] = (row max) + 1.0 after the cast, a margin
    above the bf16 spacing there, so the planted token is the strict argmax.
    p falls linearly from plant_hi at the root to plant_lo at the deepest
    internal depth.
    """
    parents = np.asarray(parents)
    tokens = np.asarray(tokens)
    batch, n = parents.shape
    dt = w.torch_dtype
    out = torch.empty((batch, n, w.vocab), dtype=dt)
    for b in range(batch):
        rows = _randn((n, w.vocab), (w.cfg_id, _T_LOG, seed, b), w.logit_sigma).to(dt)
        if plant:
            rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(
                [w.cfg_id, _T_PLANT, seed, b])))
            depth = trees.node_depths(parents[b])
            kids = {}
            for c in range(1, n):
                kids.setdefault(int(parents[b][c]), []).append(c)
            dmax = max([int(depth[v]) for v in kids] + [1])
            for v in range(n):
                u = rng.uniform()
                if v not in kids:
                    continue
                p = w.plant_hi + (w.plant_lo - w.plant_hi) * min(int(depth[v]) / dmax, 1.0)
                c = kids[v][int(rng.integers(0, len(kids[v])))]
                if u < p:
                    rowmax = float(rows[v].float().max())
                    rows[v, int(tokens[b][c])] = torch.tensor(rowmax + 1.0).to(dt)
        out[b] = rows
    return out


def round_inputs(w, seed=0, poison=False, tree_shape="best_first", variant=None):
    """Everything one round of workload ``w`` consumes, as CPU tensors."""
    ctx_lens = context_lengths(w, seed)
    res = {"workload": w, "ctx_lens": ctx_lens, "image_lens": image_lengths(w, ctx_lens, seed)}
    if "draft" in w.steps:
        res["draft"] = attention_inputs(w, "draft", w.n_draft, ctx_lens, seed, variant, poison,
                                        cap=w.cap)
    if "verify" in w.steps or "accept" in w.steps:
        par, tok = tree_inputs(w, seed, tree_shape)
        res["parents"], res["tokens"] = par, tok
    if "verify" in w.steps:
        res["verify"] = attention_inputs(w, "verify", w.n_tree, ctx_lens, seed, variant, poison,
                                         cap=w.cap)
    if "accept" in w.steps:
        res["logits"] = planted_logits(w, res["parents"], res["tokens"], seed)
    return res


def custom_workload(base, **kw):
    """A copy of a named workload with some fields replaced (for edge-case tests)."""
    return dataclasses.replace(WORKLOADS[base] if isinstance(base, str) else base, **kw)


_T_DRAFT_LOGITS, _T_DRAFT_PLANT, _T_ROOTS = 9, 10, 11


def draft_logits(w, seed=0, batch=None, horizon=None, vocab=None, variant=None, dtype=None):
    """Drafter logits [batch][L][V] at offsets j = 1..L (L = block size - 1 by default).

    The block head's rows are not available (no weights), so these mimic a
    confident drafter whose certainty fades with the offset: background logits
    ~ N(0, 1), plus at every offset four planted tokens (distinct, uniform)
    whose logits are  top_j - 1.5 r - U(0, 0.5)  for r = 0..3, with top_j falling
    linearly from 16 at j = 1 to 8 at j = L.  Against the ~log(V) + 0.5 = 12.4
    log-normaliser of the background this puts q_1(best) near 0.97 and
    q_L(best) near 0.01, so the top-63 trees reach depth 7-8 along a
    high-probability spine with side branches, as the paper's
    top-N-by-product trees do.

    variant   None, "ties" (every offset's best planted logit copied onto two
              more tokens: exact bf16/fp32 ties), "uniform" (all logits 0),
              "masked" (all but 5 tokens per offset at -inf)
    """
    batch = batch if batch is not None else w.batch
    L = horizon if horizon is not None else w.n_draft - 1
    V = vocab if vocab is not None else w.vocab
    dt = dtype if dtype is not None else w.torch_dtype
    out = torch.empty((batch, L, V), dtype=dt)
    for b in range(batch):
        if variant == "uniform":
            out[b] = 0.0
            continue
        rows = _randn((L, V), (w.cfg_id, _T_DRAFT_LOGITS, seed, b), 1.0)
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(
            [w.cfg_id, _T_DRAFT_PLANT, seed, b])))
        for j in range(L):
            top = 16.0 - 8.0 * (j / max(L - 1, 1))
            k = min(4, V)
            toks = rng.choice(V, size=min(k + 2, V), replace=False)
            for r in range(k):
                rows[j, int(toks[r])] = top - 1.5 * r - rng.uniform(0.0, 0.5)
            if variant == "ties":
                for t in toks[k:]:
                    rows[j, int(t)] = rows[j, int(toks[0])]
            if variant == "masked":
                keep = np.zeros(V, dtype=bool)
                keep[toks[:k]] = True
                keep[int(rng.integers(0, V))] = True
                rows[j, torch.as_tensor(~keep)] = float("-inf")
        out[b] = rows.to(dt)
    return out


def draft_roots(w, seed=0, batch=None, vocab=None):
    """The pending root token b of every sequence (uniform over the vocabulary)."""
    batch = batch if batch is not None else w.batch
    V = vocab if vocab is not None else w.vocab
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([w.cfg_id, _T_ROOTS, seed])))
    return torch.as_tensor(rng.integers(0, V, size=batch).astype(np.int32))
