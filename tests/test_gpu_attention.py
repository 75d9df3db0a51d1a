"""Parity of the HIP draft / verify attention with the float64 oracle.

Element-by-element on every output at oracle-sized shapes that span several
key tiles, several splits and a ragged tail; sampled rows at the full
workload sizes, in the launch configuration the benchmark times.  Inputs come
from the seeded generators in ``workloads`` and are fed unchanged to both sides.
"""

import numpy as np
import pytest
import torch

import paper_2609_00355_amd as G
from gpu_helpers import TOL, assert_close, ensure_lib, oracle_attention, run_attention
from workloads import configs as C

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_lib()


def _w(name, **kw):
    return C.custom_workload(name, **kw)


def _check(kind, w, ctx_lens, n, seed=0, variant=None, poison=False, tree_shape="best_first",
           cap=None, what="", workspace=None):
    inp = C.attention_inputs(w, kind, n, ctx_lens, seed, variant, poison, cap=cap)
    par = None
    if kind == "verify":
        par, _ = C.tree_inputs(w, seed, tree_shape, n=n, batch=len(ctx_lens))
    out, lse = run_attention(kind, inp, par, workspace=workspace)
    ref_out, ref_lse = oracle_attention(kind, inp, par)
    print(f"[{what}] {kind} n={n} ctx={list(ctx_lens)[:4]} variant={variant}", flush=True)
    return assert_close(out, lse, ref_out, ref_lse, w.dtype, what)


# ------------------------------------------------------------- fp32 (VALU path)
def test_tiny_fp32_draft_and_verify():
    w = C.WORKLOADS["tiny_fp32"]
    ctx = C.context_lengths(w)
    _check("draft", w, ctx, w.n_draft, what="tiny_fp32 draft")
    _check("verify", w, ctx, w.n_tree, what="tiny_fp32 verify")


@pytest.mark.parametrize("kind", ["draft", "verify"])
@pytest.mark.parametrize("variant", [None, "sharp1", "sharp4", "tree_dominant"])
def test_fp32_variants(kind, variant):
    w = _w("tiny_fp32")
    _check(kind, w, [300], 16, seed=1, variant=variant, poison=True, what=f"fp32 {variant}")


@pytest.mark.parametrize("d,hq,hkv", [(64, 4, 1), (128, 8, 1), (64, 6, 3), (128, 16, 2)])
@pytest.mark.parametrize("n", [1, 5, 64])
def test_fp32_shapes(d, hq, hkv, n):
    w = _w("tiny_fp32", d=d, hq=hq, hkv=hkv)
    for kind in ("draft", "verify"):
        _check(kind, w, [0, 65, 129], n, seed=2, variant="sharp1", poison=True, cap=200,
               what=f"fp32 d{d} h{hq}/{hkv}")


@pytest.mark.parametrize("shape", ["chain", "star", "best_first"])
def test_fp32_tree_shapes(shape):
    w = _w("tiny_fp32", n_tree=40, depth_cap=39)
    _check("verify", w, [77, 0], 40, seed=3, variant="tree_dominant", tree_shape=shape,
           what=f"fp32 {shape}")


# ------------------------------------------------------------- bf16 (MFMA path)
def test_draft_2k_full():
    w = C.WORKLOADS["draft_2k"]
    _check("draft", w, C.context_lengths(w), w.n_draft, what="draft_2k")


def test_verify_4k_full():
    w = C.WORKLOADS["verify_4k"]
    _check("verify", w, C.context_lengths(w), w.n_tree, what="verify_4k")


@pytest.mark.parametrize("kind", ["draft", "verify"])
@pytest.mark.parametrize("variant", ["sharp1", "sharp4", "tree_dominant"])
def test_bf16_sharp_variants(kind, variant):
    w = _w("verify_4k")
    n = 16 if kind == "draft" else 64
    _check(kind, w, [1000, 37], n, seed=4, variant=variant, poison=True, cap=1100,
           what=f"bf16 {variant}")


@pytest.mark.parametrize("n", [1, 7, 16, 33, 64])
@pytest.mark.parametrize("ctx", [[0], [1], [63, 64, 65], [700, 0, 1]])
def test_bf16_rows_and_context_edges(n, ctx):
    w = _w("verify_4k", batch=len(ctx))
    for kind in ("draft", "verify"):
        _check(kind, w, ctx, n, seed=5, variant="sharp1", poison=True, cap=max(max(ctx), 1) + 5,
               what=f"bf16 edges n={n}")


@pytest.mark.parametrize("d,hq,hkv", [(64, 28, 4), (128, 8, 1), (128, 16, 2), (128, 4, 4)])
def test_bf16_head_shapes(d, hq, hkv):
    w = _w("verify_4k", d=d, hq=hq, hkv=hkv)
    for kind in ("draft", "verify"):
        _check(kind, w, [513, 90], 24, seed=6, variant="sharp1", poison=True, cap=600,
               what=f"bf16 d{d} h{hq}/{hkv}")


@pytest.mark.parametrize("shape", ["chain", "star"])
def test_bf16_chain_and_star(shape):
    w = _w("verify_4k", n_tree=64, depth_cap=63)
    _check("verify", w, [200], 64, seed=7, variant="tree_dominant", tree_shape=shape,
           what=f"bf16 {shape}")


@pytest.mark.parametrize("v_scale", [3.0e8, 1.0e-30])
@pytest.mark.parametrize("kind", ["draft", "verify"])
def test_bf16_value_range(kind, v_scale):
    """Values far outside fp16 range, above (outputs ~ 1e8) and below
    (outputs ~ 1e-31): every intermediate of the bf16 path (probabilities, the
    fp16 split partials with their row scale, merge) must keep the range, so
    the error stays at the bf16 output's relative precision."""
    w = _w("verify_4k", batch=2)
    n = 16 if kind == "draft" else 64
    inp = C.attention_inputs(w, kind, n, [700, 90], 8, None, False, cap=800)
    for key in ("v_ctx", "v_new"):
        inp[key] = (inp[key].float() * v_scale).to(inp[key].dtype)
    par = None
    if kind == "verify":
        par, _ = C.tree_inputs(w, 8, "best_first", n=n, batch=2)
    out, lse = run_attention(kind, inp, par)
    ref_out, ref_lse = oracle_attention(kind, inp, par)
    assert np.all(np.isfinite(out))
    scale = np.abs(ref_out).max()
    err = np.abs(out - ref_out).max()
    print(f"[bf16 value range] {kind} x{v_scale:g}: max|O| {scale:.3e}, max err {err:.3e}", flush=True)
    assert (scale > 1e5) if v_scale > 1 else (0 < scale < 1e-25)
    assert err <= TOL["bf16"]["rel"] * scale, f"error {err:.3e} > {TOL['bf16']['rel']} x {scale:.3e}"
    assert np.abs(lse - ref_lse).max() <= TOL["bf16"]["lse"] * max(1.0, np.abs(ref_lse).max())


# The key pieces are planned on the device from ctx_lens: at 28/4 heads a
# sequence of ctx keys is cut into about ceil((ctx / 64 + 1) / T) pieces with
# T >= 4 tiles, so these contexts give one piece (no merge), two, a dozen and
# several dozen (draft: 64 slots per KV head, verify: 32 per row group).
@pytest.mark.parametrize("ctx", [100, 300, 3000, 20000])
def test_piece_count_invariance(ctx):
    w = _w("verify_4k", batch=1)
    for kind, n in (("draft", 16), ("verify", 64)):
        _check(kind, w, [ctx], n, seed=8, variant="sharp1", cap=ctx + 7, what=f"ctx {ctx}")


def test_many_sequences_more_than_slots():
    """40 sequences > the 32 verify slots per KV head that 256 workgroups
    would give: the plan takes one slot per sequence at least."""
    w = _w("verify_4k", batch=40)
    rng = np.random.default_rng(12)
    ctx = [int(x) for x in rng.integers(0, 700, size=40)]
    for kind, n in (("draft", 16), ("verify", 64)):
        _check(kind, w, ctx, n, seed=12, variant="sharp1", poison=True, cap=720, what="40 sequences")


def test_workspace_reuse_across_shapes():
    """One workspace serves calls of different shapes in turn: every call
    leaves its arrival counters at zero for the next."""
    w = _w("verify_4k", batch=2)
    ws = torch.zeros(64 << 20, dtype=torch.uint8, device="cuda")
    for ctx, n, kind in (([3000, 1234], 64, "verify"), ([900, 20], 16, "draft"), ([5000, 4000], 64, "verify"),
                         ([3000, 1234], 16, "draft")):
        _check(kind, w, ctx, n, seed=13, variant="sharp1", cap=5100, what=f"reuse {kind} {ctx}", workspace=ws)


def test_ragged_batch_small():
    w = _w("verify_4k", batch=6)
    ctx = [0, 1, 64, 1000, 2500, 3333]
    for kind, n in (("draft", 16), ("verify", 64)):
        _check(kind, w, ctx, n, seed=9, poison=True, cap=3400, what="ragged small")


def test_deterministic_bitwise():
    w = _w("verify_4k", batch=2)
    inp = C.attention_inputs(w, "verify", 64, [2000, 999], 10, "sharp1", cap=2100)
    par, _ = C.tree_inputs(w, 10, n=64, batch=2)
    a = run_attention("verify", inp, par)
    b = run_attention("verify", inp, par)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])


def test_explicit_scale():
    w = _w("verify_4k", batch=1)
    inp = C.attention_inputs(w, "verify", 64, [500], 11, "sharp1", cap=500)
    par, _ = C.tree_inputs(w, 11, n=64, batch=1)
    out, lse = run_attention("verify", inp, par, sm_scale=0.02)
    ref_out, ref_lse = oracle_attention("verify", inp, par, sm_scale=0.02)
    assert_close(out, lse, ref_out, ref_lse, "bf16", "explicit scale")


# ------------------------------------------------------------- full workload sizes
def _sampled_full(name, kind, seed=0):
    w = C.WORKLOADS[name]
    ctx = C.context_lengths(w, seed)
    n = w.n_draft if kind == "draft" else w.n_tree
    inp = C.attention_inputs(w, kind, n, ctx, seed, None, False, cap=w.cap)
    par = None
    if kind == "verify":
        par, _ = C.tree_inputs(w, seed)
    out, lse = run_attention(kind, inp, par)
    rows = sorted({0, 1, n // 2, n - 1})
    ref_out, ref_lse = oracle_attention(kind, inp, par, rows=rows)
    print(f"[{name} {kind}] ctx={list(ctx)[:6]} rows={rows}", flush=True)
    assert_close(out[:, rows], lse[:, rows], ref_out, ref_lse, w.dtype, f"{name} {kind} sampled")
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(lse))


@pytest.mark.parametrize("kind", ["draft", "verify"])
def test_doc_16k_full_size_sampled(kind):
    _sampled_full("doc_16k", kind)


@pytest.mark.parametrize("seed", [0, 1])
@pytest.mark.parametrize("kind", ["draft", "verify"])
def test_ragged_mix_full_size_sampled(kind, seed):
    _sampled_full("ragged_mix", kind, seed)


# Every row of the full doc_16k shapes (batch 4, 16384 context keys, 28/4
# heads) against the oracle, with sharp scores (Q, K, V ~ N(0, 1): softmax
# mass on a few keys, so a misplaced key or a wrong mask shows) and with
# tree-dominant keys (each node's own key aligned with its queries, so the
# ancestor mask decides most of the mass).  The launch configuration is the
# one the benchmark times.
@pytest.mark.parametrize("variant", ["sharp1", "tree_dominant"])
@pytest.mark.parametrize("kind", ["draft", "verify"])
def test_doc_16k_every_row(kind, variant):
    w = C.WORKLOADS["doc_16k"]
    ctx = C.context_lengths(w, 0)
    n = w.n_draft if kind == "draft" else w.n_tree
    inp = C.attention_inputs(w, kind, n, ctx, 3, variant, False, cap=w.cap)
    par = C.tree_inputs(w, 3)[0] if kind == "verify" else None
    out, lse = run_attention(kind, inp, par)
    ref_out, ref_lse = oracle_attention(kind, inp, par)
    print(f"[doc_16k every row] {kind} {variant}", flush=True)
    assert_close(out, lse, ref_out, ref_lse, w.dtype, f"doc_16k {kind} {variant} every row")


def test_ragged_mix_plan_balance():
    """The piece plan the kernels derive from the device context lengths
    (read back from the workspace: pieces and first slot per sequence) gives
    the ragged serving mix pieces whose longest is within 1.5x the mean keys
    per piece, and covers every sequence's tiles."""
    w = C.WORKLOADS["ragged_mix"]
    ctx = C.context_lengths(w, 0)
    inp = C.attention_inputs(w, "verify", w.n_tree, ctx, 0, None, False, cap=w.cap)
    par, _ = C.tree_inputs(w, 0)
    ws = torch.zeros(256 << 20, dtype=torch.uint8, device="cuda")
    run_attention("verify", inp, par, workspace=ws)
    plan = ws[: 8 * w.batch].cpu().view(torch.int32).numpy().reshape(w.batch, 2)  # (pieces, first slot)
    tiles = np.array([(int(c) + 63) // 64 + 1 for c in ctx])  # context tiles + the new-key tile
    count = plan[:, 0]
    assert np.all(count >= 1)
    # pieces of one sequence take consecutive slots, sequence after sequence
    assert plan[0, 1] == 0 and np.all(plan[1:, 1] == plan[:-1, 1] + count[:-1])
    longest = int(np.max((tiles + count - 1) // count))
    mean = tiles.sum() / count.sum()
    print(f"[ragged plan] pieces {count.tolist()} longest {longest} tiles, mean {mean:.1f}", flush=True)
    assert longest <= 1.5 * mean
