"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI
and the float64 oracle on the same seeded inputs, and compare."""

import os

import numpy as np
import torch

import paper_2609_00355_amd as G
from oracle import accept as OA
from oracle import attention as OT

# Tolerances.  Spec bounds on the output: max-abs 1e-4 for fp32 and 2e-2
# for bf16 outputs.  Because the configs' N(0,1)/sqrt(D) inputs make outputs
# tiny (|O| ~ 1e-2), a second, normalised bound is applied as well:
#   fp32: |O - O_ref| <= 2e-5 * max|O_ref|   (fp32 accumulation over <= 64k keys,
#         exp2 with ~1 ulp error; measured errors are ~1e-6 relative)
#   bf16: |O - O_ref| <= 1.5e-2 * max|O_ref| (output rounded to bf16: 2^-9 relative,
#         probabilities rounded to bf16 before P.V: 2^-9 relative each, averaging out)
# LSE is computed from fp32 scores of the exact inputs in both paths.
TOL = {
    "f32": dict(abs=1e-4, rel=2e-5, lse=1e-4),
    "bf16": dict(abs=2e-2, rel=1.5e-2, lse=2e-3),
}


def ensure_lib():
    if not os.path.exists(G.LIB_PATH):
        from paper_2609_00355_amd import build
        build.build()
    G.lib()


def to_dev(d):
    return {k: (v.cuda() if torch.is_tensor(v) else v) for k, v in d.items()}


def run_attention(kind, inp, parents=None, sm_scale=0.0, workspace=None):
    dev = to_dev(inp)
    if kind == "draft":
        out, lse = G.glance_block_draft_attn(dev["q"], dev["k_ctx"], dev["v_ctx"], dev["k_new"],
                                             dev["v_new"], dev["ctx_lens"], sm_scale=sm_scale,
                                             workspace=workspace)
    else:
        out, lse = G.glance_tree_verify_attn(dev["q"], dev["k_ctx"], dev["v_ctx"], dev["k_new"],
                                             dev["v_new"], dev["ctx_lens"], parents.cuda(),
                                             sm_scale=sm_scale, workspace=workspace)
    torch.cuda.synchronize()
    return out.float().cpu().numpy(), lse.cpu().numpy()


def oracle_attention(kind, inp, parents=None, rows=None, sm_scale=None):
    if kind == "draft":
        return OT.block_draft_attn(inp["q"], inp["k_ctx"], inp["v_ctx"], inp["k_new"], inp["v_new"],
                                   inp["ctx_lens"], sm_scale=sm_scale, rows=rows)
    return OT.tree_verify_attn(inp["q"], inp["k_ctx"], inp["v_ctx"], inp["k_new"], inp["v_new"],
                               inp["ctx_lens"], parents, sm_scale=sm_scale, rows=rows)


def assert_close(out, lse, ref_out, ref_lse, dtype, what=""):
    tol = TOL[dtype]
    assert np.all(np.isfinite(out)), f"{what}: non-finite output"
    err = np.abs(out - ref_out).max()
    scale = np.abs(ref_out).max()
    assert err <= tol["abs"], f"{what}: max-abs error {err:.3e} > {tol['abs']}"
    assert err <= tol["rel"] * scale + 1e-30, f"{what}: error {err:.3e} > {tol['rel']} x max|O_ref| {scale:.3e}"
    lerr = np.abs(lse - ref_lse).max()
    assert lerr <= tol["lse"] * max(1.0, np.abs(ref_lse).max()), f"{what}: LSE error {lerr:.3e}"
    return err, scale, lerr


def run_accept(logits, parents, tokens, path_stride=None):
    res = G.glance_greedy_accept(logits.cuda(), parents.cuda(), tokens.cuda(), path_stride=path_stride)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in res.items()}


def assert_accept_equal(got, logits, parents, tokens, path_stride=None):
    ref = OA.greedy_accept(logits, parents, tokens, path_stride=path_stride or parents.shape[1])
    np.testing.assert_array_equal(got["argmax"], ref["argmax"])
    np.testing.assert_array_equal(got["accept_len"], ref["accept_len"])
    np.testing.assert_array_equal(got["accept_path"], ref["accept_path"])
    np.testing.assert_array_equal(got["next_root"], ref["next_root"])
    return ref
