"""GPU parity of the draft tree builder (glance_build_tree) against the
float64 oracle (oracle/tree.py) on the same seeded drafter logits.

The GPU ranks strings by fp32 scores, the oracle by float64 ones, so the two
may order strings whose scores lie within rounding of each other either way.
Each case is therefore checked in two layers:

* always: the GPU tree is well formed (root, parents[i] < i, depth <= L,
  distinct siblings), every GPU score is within eps of the float64 score of
  its string, GPU scores are non-increasing, every GPU string scores at least
  the oracle's N-th best minus the rounding band, and every oracle string
  clear of the band around the (N+1)-th best is kept;
* the GPU's kept scores, sorted, equal the oracle's N best within the band
  (a near-tie may swap strings, never drop a clearly better one);
* when the oracle's N + 1 best strings are "clean" (every adjacent pair is
  either separated by more than the two rounding bands or an exact structural
  tie: the same logit at every offset, which fp32 ties exactly too), the GPU
  parents and tokens must equal the oracle's exactly.

eps for a string of length l: each of its l terms log q = z - lse carries the
fp32 rounding of lse (a sum of exp over the row, exp2/log2 within 1 ulp) plus
its own subtraction, and the left-to-right sum adds one rounding per term:
    eps(l, s) = l * (1e-5 + 2.4e-7 * (|s| + max|lse|)),
about 10 ulp of the magnitudes involved per term.
"""

import numpy as np
import pytest
import torch

import paper_2609_00355_amd as G
from oracle import tree as OT
from workloads import configs as W
from workloads import trees as WT

from gpu_helpers import ensure_lib

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_lib()


def _eps(length, score, lse_max):
    return length * (1e-5 + 2.4e-7 * (abs(score) + lse_max))


def _lse_max(z64):
    m = z64.max(axis=-1)
    with np.errstate(invalid="ignore", over="ignore"):
        lse = m + np.log(np.exp(z64 - m[:, None]).sum(axis=-1))
    lse = lse[np.isfinite(lse)]
    return float(np.abs(lse).max()) if lse.size else 0.0


def run_tree(z, roots, budget, first_row=0, horizon=None):
    out = G.glance_build_tree(z.cuda(), roots.cuda(), budget, first_row=first_row, horizon=horizon)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def _gpu_strings(par, tok):
    strings = [()]
    for i in range(1, len(par)):
        strings.append(strings[par[i]] + (int(tok[i]),))
    return strings[1:]


def check_sequence(z, root, budget, par, tok, sc):
    """Compare one sequence's GPU tree with the oracle.  Returns True if the case was clean."""
    z64 = OT._as_f64(z)
    L, V = z64.shape
    lq = OT.log_marginals(z64)
    lse_max = _lse_max(z64)
    n = budget
    # structure
    assert par[0] == -1 and tok[0] == root
    assert np.all((par[1:] >= 0) & (par[1:] < np.arange(1, n + 1)))
    depth = WT.node_depths(par)
    assert depth.max() <= L
    kids = {}
    for i in range(1, n + 1):
        kids.setdefault(int(par[i]), []).append(int(tok[i]))
    for p_, ts in kids.items():
        assert len(ts) == len(set(ts)), f"duplicate sibling tokens under node {p_}"
    g_strings = _gpu_strings(par, tok)
    sig = np.array([OT.string_score(lq, s) for s in g_strings])
    eps = np.array([_eps(len(s), x, lse_max) for s, x in zip(g_strings, sig)])
    both_inf = np.isneginf(sig) & np.isneginf(sc[1:])
    assert sc[0] == 0.0
    err = np.where(both_inf, 0.0, np.abs(sc[1:].astype(np.float64) - sig))
    assert np.all(err <= eps), f"score error {err.max():.3g} > eps"
    assert np.all(np.diff(sc[1:]) <= 0), "GPU scores must be non-increasing"
    # the oracle's best N (+1 when it exists)
    total = sum(V ** l for l in range(1, L + 1))
    ref = OT.build_tree(z64, root, min(n + 1, total))
    r_strings, r_sc = ref["strings"], ref["scores"][1:]
    r_eps = np.array([_eps(len(s), x, lse_max) for s, x in zip(r_strings, r_sc)])
    band = 2 * max(r_eps.max(), eps.max())
    s_n = r_sc[n - 1]
    if np.isfinite(s_n):
        assert np.all(sig >= s_n - band), "a GPU string scores clearly below the oracle's N-th best"
    g_set = set(g_strings)
    fin = np.isfinite(r_sc[:n])
    srt = np.sort(sig)[::-1]
    assert np.all(np.isfinite(srt) == fin)
    assert np.all(np.abs(srt[fin] - r_sc[:n][fin]) <= band), "kept scores differ from the oracle's N best"
    if len(r_strings) > n:
        s_next = r_sc[n]
        for s, x in zip(r_strings[:n], r_sc[:n]):
            if np.isfinite(x) and x > s_next + band:
                assert s in g_set, f"string {s} (score {x}) clearly in the top {n} is missing"
    # clean: exact agreement required
    zvals = [tuple(z64[j, t] for j, t in enumerate(s)) for s in r_strings]
    clean = True
    for i in range(len(r_strings) - 1):
        if zvals[i] == zvals[i + 1] and len(r_strings[i]) == len(r_strings[i + 1]):
            continue
        a, b = r_sc[i], r_sc[i + 1]
        if np.isneginf(a) and np.isneginf(b):
            continue
        if not (a - b > r_eps[i] + r_eps[i + 1]):
            clean = False
            break
    if clean:
        np.testing.assert_array_equal(par, ref["parents"][:n + 1])
        np.testing.assert_array_equal(tok, ref["tokens"][:n + 1])
    return clean


def check_batch(z, roots, budget, out):
    cleans = []
    for b in range(z.shape[0]):
        cleans.append(check_sequence(z[b], int(roots[b]), budget, out["parents"][b], out["tokens"][b],
                                     out["scores"][b]))
    return cleans


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("budget", [1, 15, 63])
def test_small_vocab(dtype, budget):
    w = W.WORKLOADS["tiny_fp32"]
    z = W.draft_logits(w, seed=budget, batch=2, horizon=6, vocab=1000, dtype=dtype)
    roots = W.draft_roots(w, seed=budget, batch=2, vocab=1000)
    out = run_tree(z, roots, budget)
    cleans = check_batch(z, roots, budget, out)
    # bf16 logits lie on a coarse grid, so distinct strings often tie exactly
    # in real arithmetic and rounding decides; fp32 ones do not
    if dtype == torch.float32:
        assert all(cleans)


@pytest.mark.parametrize("seed", [0, 1])
def test_doc_16k_draft_rows(seed):
    """Full size: batch 4, 15 offsets of a 152064-token vocabulary, bf16, budget 63."""
    w = W.WORKLOADS["doc_16k"]
    z = W.draft_logits(w, seed=seed)
    roots = W.draft_roots(w, seed=seed)
    out = run_tree(z, roots, 63)
    check_batch(z, roots, 63, out)


def test_doc_16k_shapes_fp32_exact():
    """Full vocabulary in fp32 (no grid ties): the trees must equal the oracle's."""
    w = W.WORKLOADS["doc_16k"]
    z = W.draft_logits(w, seed=2, dtype=torch.float32)
    roots = W.draft_roots(w, seed=2)
    out = run_tree(z, roots, 63)
    assert sum(check_batch(z, roots, 63, out)) >= 3


def test_block_head_rows_with_root_row_skipped():
    """[batch][B][V] rows with row 0 (the root's) skipped: pointer + V, stride B * V."""
    w = W.WORKLOADS["doc_16k"]
    z = W.draft_logits(w, seed=3, batch=2, horizon=16)
    roots = W.draft_roots(w, seed=3, batch=2)
    out = run_tree(z, roots, 63, first_row=1)
    check_batch(z[:, 1:].contiguous(), roots, 63, out)
    out2 = run_tree(z[:, 1:].contiguous(), roots, 63)
    for k in ("parents", "tokens", "scores"):
        np.testing.assert_array_equal(out[k], out2[k])


@pytest.mark.parametrize("variant", ["ties", "masked"])
def test_tie_and_masked_rows(variant):
    w = W.WORKLOADS["doc_16k"]
    z = W.draft_logits(w, seed=4, batch=2, variant=variant)
    roots = W.draft_roots(w, seed=4, batch=2)
    out = run_tree(z, roots, 63)
    check_batch(z, roots, 63, out)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_clustered_slice_takes_the_exact_fallback(dtype):
    """Twenty of the row's best values in one 1024-value slice, five in each of
    its four 16-lane rows: the slice keeps only the values at or above the
    smallest row maximum (16 of them), so four of the row's best are left out
    and the ranking pass must see that and select exactly from the whole row."""
    g = torch.Generator().manual_seed(11)
    z = torch.randn(1, 3, 152064, generator=g)
    vpl = 8 if dtype == torch.bfloat16 else 4         # values per 16-byte load
    for r in range(4):
        for i in range(5):
            z[0, 0, r * 16 * vpl + i * vpl] = 20.0 - 0.125 * (5 * r + i)
    z = z.to(dtype)
    roots = torch.tensor([5], dtype=torch.int32)
    out = run_tree(z, roots, 63)
    clean = check_batch(z, roots, 63, out)
    if dtype == torch.float32:
        assert clean == [True]
    # all twenty planted tokens of the first offset are one-token strings
    one_tok = {int(t) for p_, t in zip(out["parents"][0, 1:], out["tokens"][0, 1:]) if p_ == 0}
    assert {r * 16 * vpl + i * vpl for r in range(4) for i in range(5)} <= one_tok


@pytest.mark.parametrize("vocab", [3000, 152064])
def test_uniform_rows_take_the_exact_fallback(vocab):
    """All logits equal: every value reaches the candidate list, which overflows
    for these sizes, so the exact radix selection runs; ties go by index."""
    w = W.WORKLOADS["doc_16k"]
    z = W.draft_logits(w, batch=1, horizon=4, vocab=vocab, variant="uniform")
    roots = torch.tensor([7], dtype=torch.int32)
    out = run_tree(z, roots, 63)
    assert check_batch(z, roots, 63, out) == [True]
    assert out["tokens"][0, 1:].tolist() == list(range(63))     # 63 one-token strings, index order


@pytest.mark.parametrize("vocab,horizon,budget", [(5, 4, 63), (1, 15, 15), (2, 6, 63), (63, 1, 63),
                                                  (64, 2, 63), (1001, 3, 40)])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_small_and_odd_shapes(vocab, horizon, budget, dtype):
    w = W.WORKLOADS["tiny_fp32"]
    z = W.draft_logits(w, seed=vocab, batch=2, horizon=horizon, vocab=vocab, dtype=dtype)
    roots = W.draft_roots(w, seed=vocab, batch=2, vocab=vocab)
    out = run_tree(z, roots, budget)
    check_batch(z, roots, budget, out)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_vocabulary_beyond_one_slice_per_thread(dtype):
    """300001 tokens: 293 slices of 1024 values, more than the ranking pass's
    256 threads, so its loops over slices take a second round (and the last
    slice is ragged)."""
    w = W.WORKLOADS["tiny_fp32"]
    z = W.draft_logits(w, seed=7, batch=2, horizon=3, vocab=300001, dtype=dtype)
    roots = W.draft_roots(w, seed=7, batch=2, vocab=300001)
    out = run_tree(z, roots, 63)
    cleans = check_batch(z, roots, 63, out)
    if dtype == torch.float32:
        assert all(cleans)


@pytest.mark.parametrize("case", range(24))
def test_seeded_sweep(case):
    """Random shapes and value patterns (seeded): vocabularies from 3 to 70000,
    1 to 15 offsets, budgets 1 to 63, fp32 and bf16, Gaussian rows with some
    best values clustered into one 1024-value slice (the re-read path), some
    rows with coarse integer logits (ties), and some masked to -inf."""
    rng = np.random.default_rng(1000 + case)
    vocab = int(rng.choice([3, 17, 130, 1000, 4099, 20000, 70000]))
    horizon = int(rng.integers(1, 16))
    budget = int(rng.integers(1, 64))
    total = sum(vocab ** l for l in range(1, horizon + 1))
    budget = min(budget, total)
    dtype = torch.bfloat16 if case % 2 else torch.float32
    batch = int(rng.integers(1, 4))
    z = rng.normal(size=(batch, horizon, vocab))
    for b in range(batch):
        for j in range(horizon):
            kind = rng.integers(0, 4)
            if kind == 1 and vocab >= 1024:      # clustered best values in one slice
                s0 = 1024 * int(rng.integers(0, vocab // 1024))
                idx = s0 + rng.choice(1024, size=min(40, 1024), replace=False)
                z[b, j, idx] = 6.0 + rng.normal(size=idx.size)
            elif kind == 2:                       # coarse grid: exact ties
                z[b, j] = np.round(z[b, j] * 2) / 2
            elif kind == 3 and vocab > 5:         # mostly masked
                keep = rng.choice(vocab, size=max(1, vocab // 7), replace=False)
                m = np.full(vocab, -np.inf)
                m[keep] = z[b, j, keep]
                z[b, j] = m
    z = torch.from_numpy(z.astype(np.float32)).to(dtype)
    roots = torch.from_numpy(rng.integers(0, vocab, size=batch).astype(np.int32))
    out = run_tree(z, roots, budget)
    check_batch(z, roots, budget, out)


def test_row_of_minus_inf():
    z = torch.randn(1, 5, 700, generator=torch.Generator().manual_seed(3))
    z[0, 2] = float("-inf")
    roots = torch.tensor([1], dtype=torch.int32)
    out = run_tree(z, roots, 63)
    check_batch(z, roots, 63, out)


def test_many_sequences():
    w = W.WORKLOADS["ragged_mix"]
    z = W.draft_logits(w, seed=0)
    roots = W.draft_roots(w, seed=0)
    out = run_tree(z, roots, 63)
    check_batch(z, roots, 63, out)


def test_repeated_calls_reuse_the_workspace():
    w = W.WORKLOADS["doc_16k"]
    z1 = W.draft_logits(w, seed=5, batch=2).cuda()
    z2 = W.draft_logits(w, seed=6, batch=2).cuda()
    roots = W.draft_roots(w, seed=5, batch=2).cuda()
    ws = torch.empty(G.glance_tree_workspace_size(2, 15, w.vocab, 63), dtype=torch.uint8, device="cuda")
    a1 = {k: v.clone() for k, v in G.glance_build_tree(z1, roots, 63, workspace=ws).items()}
    a2 = {k: v.clone() for k, v in G.glance_build_tree(z2, roots, 63, workspace=ws).items()}
    b1 = G.glance_build_tree(z1, roots, 63, workspace=ws)
    torch.cuda.synchronize()
    for k in ("parents", "tokens", "scores"):
        assert torch.equal(a1[k], b1[k])
    assert not torch.equal(a1["tokens"], a2["tokens"])
