"""The allocation-free greedy acceptance (glance_greedy_accept_noalloc, the
static per-GPU scratch) against glance_greedy_accept (caller workspace):
argmax, accepted length, path and bonus token bit for bit, on two calls in a
row through the C ABI, the second with a smaller input, so that the second
reads nothing the first left in the shared buffer."""

import ctypes

import numpy as np
import pytest
import torch

import paper_2609_00355_amd as G
from gpu_helpers import ensure_lib
from workloads import configs as C

pytestmark = pytest.mark.gpu


def _p(t):
    return ctypes.c_void_p(t.data_ptr())


def _case(name, batch, n, vocab, seed):
    w = C.custom_workload(name, batch=batch, n_tree=n, depth_cap=min(15, n - 1), vocab=vocab)
    par, tok = C.tree_inputs(w, seed)
    logits = C.planted_logits(w, par, tok, seed)
    return logits.cuda(), par.cuda(), tok.cuda()


def _noalloc(lib, logits, par, tok, path_stride):
    batch, n, vocab = logits.shape
    out = {k: torch.full(s, -7, dtype=torch.int32, device="cuda")
           for k, s in (("argmax", (batch, n)), ("accept_len", (batch,)), ("accept_path", (batch, path_stride)),
                        ("next_root", (batch,)))}
    code = G.GLANCE_BF16 if logits.dtype == torch.bfloat16 else G.GLANCE_F32
    st = lib.glance_greedy_accept_noalloc(batch, n, vocab, code, _p(logits), _p(par), _p(tok), _p(out["argmax"]),
                                          _p(out["accept_len"]), _p(out["accept_path"]), path_stride,
                                          _p(out["next_root"]), ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == G.GLANCE_OK, G.glance_last_error()
    return out


def test_noalloc_matches_workspace_entry_point():
    ensure_lib()
    lib = G.lib()
    cases = [("verify_4k", 4, 64, 152064, 31), ("verify_4k", 2, 16, 5000, 32)]  # the second is smaller
    for name, batch, n, vocab, seed in cases:
        logits, par, tok = _case(name, batch, n, vocab, seed)
        print(f"[no-alloc] batch {batch} n {n} vocab {vocab}", flush=True)
        got = _noalloc(lib, logits, par, tok, 16)
        ref = G.glance_greedy_accept(logits, par, tok, path_stride=16)
        torch.cuda.synchronize()
        for k in ("argmax", "accept_len", "accept_path", "next_root"):
            np.testing.assert_array_equal(got[k].cpu().numpy(), ref[k].cpu().numpy(), err_msg=k)
    # fp32 logits too, after the bf16 calls
    w = C.WORKLOADS["tiny_fp32"]
    par, tok = C.tree_inputs(w, 3)
    logits = C.planted_logits(w, par, tok, 3)
    got = _noalloc(lib, logits.cuda(), par.cuda(), tok.cuda(), 8)
    ref = G.glance_greedy_accept(logits.cuda(), par.cuda(), tok.cuda(), path_stride=8)
    torch.cuda.synchronize()
    for k in ("argmax", "accept_len", "accept_path", "next_root"):
        np.testing.assert_array_equal(got[k].cpu().numpy(), ref[k].cpu().numpy(), err_msg=k)
