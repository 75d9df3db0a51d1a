"""Python binding of libglance.so, the GLANCE decode-round hot path on MI355X.

Thin ctypes marshalling over the C ABI declared in include/glance.h: each
function takes torch tensors that already live on the GPU, checks their
dtype, layout and shape, and passes raw device pointers plus the current HIP
stream to the library.  Outputs and workspaces the caller does not supply are
allocated with torch (device memory plumbing); every step of the computation
runs in the library's HIP kernels.  There is no fallback: if the library is
missing or a GPU is absent, the calls raise.

    glance_block_draft_attn(q, k_ctx, v_ctx, k_new, v_new, ctx_lens) -> (out, lse)
    glance_tree_verify_attn(q, k_ctx, v_ctx, k_new, v_new, ctx_lens, parents) -> (out, lse)
    glance_greedy_accept(logits, parents, tokens) -> dict(argmax, accept_len, accept_path, next_root)
    glance_sample_accept(logits, parents, tokens, temperature, seed, round_)
        -> dict(draws, accept_len, accept_path, next_root)
    glance_build_tree(draft_logits, roots, budget) -> dict(parents, tokens, scores)
    glance_commit_path(k_new, v_new, accept_len, accept_path, k_ctx, v_ctx, ctx_lens)  (in place)

Layouts: q, out [batch][n][Hq][D]; k_ctx, v_ctx [batch][Hkv][capacity][D];
k_new, v_new [batch][n][Hkv][D]; ctx_lens [batch] int32; parents, tokens
[batch][n] int32; logits [batch][n][vocab]; draft_logits [batch][rows][vocab]
(rows first_row .. first_row + horizon - 1 are the drafter's offsets 1..L).
"""

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libglance.so")

GLANCE_OK, GLANCE_ERR_INVALID_ARG, GLANCE_ERR_UNSUPPORTED, GLANCE_ERR_WORKSPACE, GLANCE_ERR_HIP = \
    0, -1, -2, -3, -4
GLANCE_F32, GLANCE_BF16 = 0, 1


class GlanceError(RuntimeError):
    def __init__(self, status, detail):
        super().__init__(f"{detail} (status {status})")
        self.status = status


class AttnShape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_new", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("ctx_capacity", ctypes.c_int32), ("sm_scale", ctypes.c_float),
                ("dtype", ctypes.c_int)]


_lib = None
_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_SZ = ctypes.c_size_t

_SIGS = {
    "glance_block_draft_attn": (ctypes.c_int, [ctypes.POINTER(AttnShape), _P, _P, _P, _P, _P, _P, _P, _P,
                                               _P, _SZ, _P]),
    "glance_tree_verify_attn": (ctypes.c_int, [ctypes.POINTER(AttnShape), _P, _P, _P, _P, _P, _P, _P, _P,
                                               _P, _P, _SZ, _P]),
    "glance_greedy_accept": (ctypes.c_int, [_I32, _I32, _I32, ctypes.c_int, _P, _P, _P, _P, _P, _P, _I32,
                                            _P, _P, _SZ, _P]),
    "glance_greedy_accept_entropy": (ctypes.c_int, [_I32, _I32, _I32, ctypes.c_int, _P, _P, _P, _P, _P, _P,
                                                    _I32, _P, _P, _P, _SZ, _P]),
    "glance_greedy_accept_noalloc": (ctypes.c_int, [_I32, _I32, _I32, ctypes.c_int, _P, _P, _P, _P, _P, _P, _I32,
                                                    _P, _P]),
    "glance_sample_accept": (ctypes.c_int, [_I32, _I32, _I32, ctypes.c_int, _P, _P, _P, ctypes.c_float,
                                            ctypes.c_uint64, ctypes.c_uint32, _P, _P, _P, _P, _I32, _P, _P,
                                            _SZ, _P]),
    "glance_build_tree": (ctypes.c_int, [_I32, _I32, _I32, _I32, ctypes.c_int, _P, ctypes.c_int64, _P, _P,
                                         _P, _P, _P, _SZ, _P]),
    "glance_tree_workspace_size": (_SZ, [_I32, _I32, _I32, _I32]),
    "glance_commit_path": (ctypes.c_int, [_I32, _I32, _I32, _I32, _I32, ctypes.c_int, _P, _P, _P, _P, _I32, _P,
                                          _P, _P, _P]),
    "glance_attn_workspace_size": (_SZ, [ctypes.POINTER(AttnShape), ctypes.c_int]),
    "glance_accept_workspace_size": (_SZ, [_I32, _I32, _I32]),
    "glance_validate_tree": (ctypes.c_int, [_I32, _P, _P, _I32]),
    "glance_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "glance_last_error": (ctypes.c_char_p, []),
    "glance_set_kernel_events": (ctypes.c_int, [_P, _P]),
    "glance_version": (_I32, []),
}


def lib():
    """Load libglance.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_00355_amd.build`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def _check(status):
    if status != GLANCE_OK:
        raise GlanceError(status, lib().glance_last_error().decode())


def glance_status_string(status):
    return lib().glance_status_string(int(status)).decode()


def glance_last_error():
    return lib().glance_last_error().decode()


def glance_version():
    return int(lib().glance_version())


def glance_validate_tree(parents, tokens=None, max_depth=-1):
    """Host check of one tree (Def. 1).  Returns (ok, message)."""
    import numpy as np
    par = np.ascontiguousarray(np.asarray(parents, dtype=np.int32))
    tok = None if tokens is None else np.ascontiguousarray(np.asarray(tokens, dtype=np.int32))
    st = lib().glance_validate_tree(int(par.size), par.ctypes.data,
                                    None if tok is None else tok.ctypes.data, int(max_depth))
    return st == GLANCE_OK, ("" if st == GLANCE_OK else glance_last_error())


def attn_shape(batch, n_new, n_q_heads, n_kv_heads, head_dim, ctx_capacity, dtype, sm_scale=0.0):
    return AttnShape(int(batch), int(n_new), int(n_q_heads), int(n_kv_heads), int(head_dim),
                     int(ctx_capacity), float(sm_scale), int(dtype))


def glance_attn_workspace_size(shape, is_verify=0):
    return int(lib().glance_attn_workspace_size(ctypes.byref(shape), int(is_verify)))


def glance_accept_workspace_size(batch, n_nodes, vocab):
    return int(lib().glance_accept_workspace_size(int(batch), int(n_nodes), int(vocab)))


def glance_tree_workspace_size(batch, horizon, vocab, budget):
    return int(lib().glance_tree_workspace_size(int(batch), int(horizon), int(vocab), int(budget)))


def glance_set_kernel_events(start, stop):
    """Record torch.cuda.Event pair around the next call's main kernel (None, None clears)."""
    a = None if start is None else ctypes.c_void_p(start.cuda_event)
    b = None if stop is None else ctypes.c_void_p(stop.cuda_event)
    _check(lib().glance_set_kernel_events(a, b))


# ---------------------------------------------------------------- tensor helpers
def _torch():
    import torch
    return torch


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.float32:
        return GLANCE_F32
    if t.dtype == torch.bfloat16:
        return GLANCE_BF16
    raise TypeError(f"unsupported dtype {t.dtype}: use float32 or bfloat16")


def _dev(t, name, dtype=None, ndim=None):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims, got shape {tuple(t.shape)}")
    return t


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _workspace(nbytes, device, workspace, stream=None):
    """The caller's workspace, or a new one allocated on the stream the call
    runs on, so that the caching allocator does not hand it to other work
    while the call's kernels still use it."""
    torch = _torch()
    if workspace is not None:
        return workspace
    # 256-byte aligned by the caching allocator
    if stream is not None and stream != torch.cuda.current_stream(device):
        with torch.cuda.stream(stream):
            return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)


def _new_output(make, like, stream, **kw):
    """A new output tensor, allocated on the stream the call runs on."""
    torch = _torch()
    if stream is not None and stream != torch.cuda.current_stream():
        with torch.cuda.stream(stream):
            return make(like, **kw)
    return make(like, **kw)


def _attn(tree, q, k_ctx, v_ctx, k_new, v_new, ctx_lens, parents, out, lse, workspace, sm_scale,
          stream, want_lse):
    torch = _torch()
    _dev(q, "q", ndim=4)
    dt = q.dtype
    code = _dtype_code(q)
    batch, n, hq, d = q.shape
    _dev(k_new, "k_new", dt, 4)
    _dev(v_new, "v_new", dt, 4)
    hkv = k_new.shape[2]
    if tuple(k_new.shape) != (batch, n, hkv, d) or tuple(v_new.shape) != (batch, n, hkv, d):
        raise ValueError("k_new / v_new must be [batch][n][Hkv][D] matching q")
    if k_ctx is not None and k_ctx.numel() > 0:
        _dev(k_ctx, "k_ctx", dt, 4)
        _dev(v_ctx, "v_ctx", dt, 4)
        cap = k_ctx.shape[2]
        if tuple(k_ctx.shape) != (batch, hkv, cap, d) or tuple(v_ctx.shape) != (batch, hkv, cap, d):
            raise ValueError("k_ctx / v_ctx must be [batch][Hkv][capacity][D]")
    else:
        cap, k_ctx, v_ctx = 0, None, None
    _dev(ctx_lens, "ctx_lens", torch.int32, 1)
    if ctx_lens.shape[0] != batch:
        raise ValueError("ctx_lens must have one entry per sequence")
    if tree:
        _dev(parents, "parents", torch.int32, 2)
        if tuple(parents.shape) != (batch, n):
            raise ValueError("parents must be [batch][n]")
    shape = attn_shape(batch, n, hq, hkv, d, cap, code, sm_scale)
    if out is None:
        out = _new_output(torch.empty_like, q, stream)
    else:
        _dev(out, "out", dt, 4)
    if lse is None and want_lse:
        lse = _new_output(torch.empty, (batch, n, hq), stream, dtype=torch.float32, device=q.device)
    elif lse is not None:
        _dev(lse, "lse", torch.float32, 3)
    need = glance_attn_workspace_size(shape, int(tree))
    if need == 0:
        raise GlanceError(GLANCE_ERR_INVALID_ARG, glance_last_error())
    ws = _workspace(need, q.device, workspace, stream)
    common = [ctypes.byref(shape), _ptr(q), _ptr(k_ctx), _ptr(v_ctx), _ptr(k_new), _ptr(v_new),
              _ptr(ctx_lens)]
    if tree:
        st = lib().glance_tree_verify_attn(*common, _ptr(parents), _ptr(out), _ptr(lse), _ptr(ws),
                                           ws.numel() * ws.element_size(), _stream(stream))
    else:
        st = lib().glance_block_draft_attn(*common, _ptr(out), _ptr(lse), _ptr(ws),
                                           ws.numel() * ws.element_size(), _stream(stream))
    _check(st)
    return out, lse


def glance_block_draft_attn(q, k_ctx, v_ctx, k_new, v_new, ctx_lens, out=None, lse=None, workspace=None,
                            sm_scale=0.0, stream=None, want_lse=True):
    """Block-draft attention (bidirectional block over the cached context).  Returns (out, lse)."""
    return _attn(False, q, k_ctx, v_ctx, k_new, v_new, ctx_lens, None, out, lse, workspace, sm_scale,
                 stream, want_lse)


def glance_tree_verify_attn(q, k_ctx, v_ctx, k_new, v_new, ctx_lens, parents, out=None, lse=None,
                            workspace=None, sm_scale=0.0, stream=None, want_lse=True):
    """Ancestor-masked tree-verify attention.  Returns (out, lse)."""
    return _attn(True, q, k_ctx, v_ctx, k_new, v_new, ctx_lens, parents, out, lse, workspace, sm_scale,
                 stream, want_lse)


def glance_greedy_accept(logits, parents, tokens, path_stride=None, outputs=None, workspace=None,
                         stream=None, want_entropy=False):
    """Row argmax + the walk of Algorithm 1.  Returns a dict of GPU tensors (int32, and
    float32 root_entropy [batch] when want_entropy, which calls
    glance_greedy_accept_entropy)."""
    args, outputs, _ = _accept_args(logits, parents, tokens, path_stride, outputs, workspace, stream,
                                    want_entropy)
    _check(_accept_fn(want_entropy)(*args))
    return outputs


def _accept_fn(want_entropy):
    return lib().glance_greedy_accept_entropy if want_entropy else lib().glance_greedy_accept


def _accept_common(logits, parents, tokens, path_stride, outputs, workspace, rows_key, stream):
    """Checks and outputs shared by both acceptances; `rows_key` names the per-row output."""
    torch = _torch()
    _dev(logits, "logits", ndim=3)
    code = _dtype_code(logits)
    batch, n, vocab = logits.shape
    _dev(parents, "parents", torch.int32, 2)
    _dev(tokens, "tokens", torch.int32, 2)
    if tuple(parents.shape) != (batch, n) or tuple(tokens.shape) != (batch, n):
        raise ValueError("parents / tokens must be [batch][n_nodes]")
    path_stride = int(path_stride or n)
    dev = logits.device
    if outputs is None:
        def new(shape):
            return _new_output(torch.empty, shape, stream, dtype=torch.int32, device=dev)
        outputs = {rows_key: new((batch, n)), "accept_len": new((batch,)), "accept_path": new((batch, path_stride)),
                   "next_root": new((batch,))}
    need = glance_accept_workspace_size(batch, n, vocab)
    if need == 0:
        raise GlanceError(GLANCE_ERR_INVALID_ARG, glance_last_error())
    ws = _workspace(need, dev, workspace, stream)
    head = [ctypes.c_int32(batch), ctypes.c_int32(n), ctypes.c_int32(vocab), ctypes.c_int(code), _ptr(logits),
            _ptr(parents), _ptr(tokens)]
    walk = [_ptr(outputs["accept_len"]), _ptr(outputs["accept_path"]), ctypes.c_int32(path_stride),
            _ptr(outputs["next_root"])]
    tail = [_ptr(ws), ctypes.c_size_t(ws.numel() * ws.element_size())]
    return head, walk, tail, outputs, ws


def _accept_args(logits, parents, tokens, path_stride, outputs, workspace, stream, want_entropy):
    torch = _torch()
    head, walk, tail, outputs, ws = _accept_common(logits, parents, tokens, path_stride, outputs, workspace,
                                                   "argmax", stream)
    if want_entropy and outputs.get("root_entropy") is None:
        outputs["root_entropy"] = _new_output(torch.empty, (logits.shape[0],), stream, dtype=torch.float32,
                                              device=logits.device)
    entropy = [_ptr(outputs["root_entropy"])] if want_entropy else []
    args = head + [_ptr(outputs["argmax"])] + walk + entropy + tail + [_stream(stream)]
    return args, outputs, ws


def glance_sample_accept(logits, parents, tokens, temperature, seed, round_, path_stride=None, outputs=None,
                         workspace=None, stream=None, round_counter=None):
    """Row draws from softmax(z / temperature) (Gumbel-max over Philox4x32-10
    noise keyed by seed, counted by round) + the walk of Algorithm 1 over the
    draws.  Returns a dict of int32 GPU tensors: draws, accept_len,
    accept_path, next_root.  round_counter: optional one-element int32 GPU
    tensor read as unsigned; the round used is round_ + its value, and the
    call advances it by one (for graph replays that draw fresh noise)."""
    args, outputs = _sample_args(logits, parents, tokens, temperature, seed, round_, path_stride, outputs,
                                 workspace, stream, round_counter)
    _check(lib().glance_sample_accept(*args))
    return outputs


def _sample_args(logits, parents, tokens, temperature, seed, round_, path_stride, outputs, workspace, stream,
                 round_counter=None):
    torch = _torch()
    seed, round_ = int(seed), int(round_)
    if not 0 <= seed < 2 ** 64 or not 0 <= round_ < 2 ** 32:
        raise ValueError("seed must fit 64 bits and round_ 32 bits, both unsigned")
    if round_counter is not None:
        _dev(round_counter, "round_counter", torch.int32, 1)
        if round_counter.numel() != 1:
            raise ValueError("round_counter must hold one element")
    head, walk, tail, outputs, _ = _accept_common(logits, parents, tokens, path_stride, outputs, workspace,
                                                  "draws", stream)
    args = head + [ctypes.c_float(float(temperature)), ctypes.c_uint64(seed), ctypes.c_uint32(round_),
                   _ptr(round_counter), _ptr(outputs["draws"])] + walk + tail + [_stream(stream)]
    return args, outputs


def _tree_args(draft_logits, roots, budget, first_row, horizon, outputs, workspace, stream, want_scores):
    torch = _torch()
    _dev(draft_logits, "draft_logits", ndim=3)
    code = _dtype_code(draft_logits)
    batch, rows, vocab = draft_logits.shape
    first_row = int(first_row)
    horizon = int(horizon if horizon is not None else rows - first_row)
    if first_row < 0 or horizon < 1 or first_row + horizon > rows:
        raise ValueError(f"rows {first_row}..{first_row + horizon - 1} are not in draft_logits' {rows} rows")
    _dev(roots, "roots", torch.int32, 1)
    if roots.shape[0] != batch:
        raise ValueError("roots must have one entry per sequence")
    dev = draft_logits.device
    n = int(budget) + 1
    if outputs is None:
        def new(dt):
            return _new_output(torch.empty, (batch, n), stream, dtype=dt, device=dev)
        outputs = {"parents": new(torch.int32), "tokens": new(torch.int32),
                   "scores": new(torch.float32) if want_scores else None}
    for name, dt in (("parents", torch.int32), ("tokens", torch.int32), ("scores", torch.float32)):
        t = outputs.get(name)
        if t is not None:
            _dev(t, name, dt, 2)
            if tuple(t.shape) != (batch, n):
                raise ValueError(f"{name} must be [batch][budget + 1]")
    need = glance_tree_workspace_size(batch, horizon, vocab, budget)
    if need == 0:
        raise GlanceError(GLANCE_ERR_INVALID_ARG, glance_last_error())
    ws = _workspace(need, dev, workspace, stream)
    base = ctypes.c_void_p(draft_logits.data_ptr() + first_row * vocab * draft_logits.element_size())
    args = [ctypes.c_int32(batch), ctypes.c_int32(horizon), ctypes.c_int32(vocab), ctypes.c_int32(int(budget)),
            ctypes.c_int(code), base, ctypes.c_int64(rows * vocab), _ptr(roots), _ptr(outputs["parents"]),
            _ptr(outputs["tokens"]), _ptr(outputs.get("scores")), _ptr(ws),
            ctypes.c_size_t(ws.numel() * ws.element_size()), _stream(stream)]
    return args, outputs, ws


def glance_build_tree(draft_logits, roots, budget, first_row=0, horizon=None, outputs=None, workspace=None,
                      stream=None, want_scores=True):
    """The budget-N draft tree of Algorithm 1's second step.

    draft_logits [batch][rows][vocab]: rows first_row .. first_row + horizon - 1
    are the drafter's offsets 1..L (first_row=1 skips the root row of a block
    head's output).  roots [batch] int32.  Returns a dict of GPU tensors
    parents, tokens [batch][budget + 1] int32 and scores [batch][budget + 1]
    float32 (None if want_scores is False).
    """
    args, outputs, _ = _tree_args(draft_logits, roots, budget, first_row, horizon, outputs, workspace, stream,
                                  want_scores)
    _check(lib().glance_build_tree(*args))
    return outputs


def _commit_args(k_new, v_new, accept_len, accept_path, k_ctx, v_ctx, ctx_lens, stream):
    torch = _torch()
    _dev(k_new, "k_new", ndim=4)
    code = _dtype_code(k_new)
    batch, n, hkv, d = k_new.shape
    _dev(v_new, "v_new", k_new.dtype, 4)
    _dev(k_ctx, "k_ctx", k_new.dtype, 4)
    _dev(v_ctx, "v_ctx", k_new.dtype, 4)
    cap = k_ctx.shape[2]
    if tuple(v_new.shape) != tuple(k_new.shape):
        raise ValueError("v_new must match k_new")
    if tuple(k_ctx.shape) != (batch, hkv, cap, d) or tuple(v_ctx.shape) != (batch, hkv, cap, d):
        raise ValueError("k_ctx / v_ctx must be [batch][Hkv][capacity][D] matching k_new")
    _dev(accept_len, "accept_len", torch.int32, 1)
    _dev(accept_path, "accept_path", torch.int32, 2)
    _dev(ctx_lens, "ctx_lens", torch.int32, 1)
    if accept_len.shape[0] != batch or accept_path.shape[0] != batch or ctx_lens.shape[0] != batch:
        raise ValueError("accept_len, accept_path and ctx_lens need one row per sequence")
    return [ctypes.c_int32(batch), ctypes.c_int32(n), ctypes.c_int32(hkv), ctypes.c_int32(d), ctypes.c_int32(cap),
            ctypes.c_int(code), _ptr(k_new), _ptr(v_new), _ptr(accept_len), _ptr(accept_path),
            ctypes.c_int32(accept_path.shape[1]), _ptr(k_ctx), _ptr(v_ctx), _ptr(ctx_lens), _stream(stream)]


def glance_commit_path(k_new, v_new, accept_len, accept_path, k_ctx, v_ctx, ctx_lens, stream=None):
    """Append the accepted path's key/value rows to the caches and advance ctx_lens (in place)."""
    _check(lib().glance_commit_path(*_commit_args(k_new, v_new, accept_len, accept_path, k_ctx, v_ctx,
                                                  ctx_lens, stream)))


# ---------------------------------------------------------------- prepared calls
class PreparedCall:
    """A library call with all arguments checked and marshalled once.

    Calling it re-issues the same C call (same pointers, same stream) with no
    per-call Python argument processing, for launch loops and graph capture.
    The tensors it references are kept alive by the object.
    """

    def __init__(self, fn, args, keep):
        self._fn = fn
        self._args = args
        self._keep = keep

    def __call__(self):
        st = self._fn(*self._args)
        if st != GLANCE_OK:
            raise GlanceError(st, glance_last_error())


def _prepare_attn(tree, q, k_ctx, v_ctx, k_new, v_new, ctx_lens, parents, out, lse, workspace, sm_scale,
                  stream):
    batch, n, hq, d = q.shape
    hkv = k_new.shape[2]
    cap = 0 if (k_ctx is None or k_ctx.numel() == 0) else k_ctx.shape[2]
    shape = attn_shape(batch, n, hq, hkv, d, cap, _dtype_code(q), sm_scale)
    ws = _workspace(glance_attn_workspace_size(shape, int(tree)), q.device, workspace, stream)
    # one checked call establishes outputs and validates everything; then freeze the arguments
    out, lse = _attn(tree, q, k_ctx, v_ctx, k_new, v_new, ctx_lens, parents, out, lse, ws,
                     sm_scale, stream, lse is not None)
    if cap == 0:
        k_ctx = v_ctx = None
    args = [ctypes.byref(shape), _ptr(q), _ptr(k_ctx), _ptr(v_ctx), _ptr(k_new), _ptr(v_new),
            _ptr(ctx_lens)]
    if tree:
        args += [_ptr(parents)]
    args += [_ptr(out), _ptr(lse), _ptr(ws), ctypes.c_size_t(ws.numel() * ws.element_size()),
             _stream(stream)]
    fn = lib().glance_tree_verify_attn if tree else lib().glance_block_draft_attn
    keep = (shape, q, k_ctx, v_ctx, k_new, v_new, ctx_lens, parents, out, lse, ws)
    return PreparedCall(fn, args, keep), out, lse


def prepare_block_draft_attn(q, k_ctx, v_ctx, k_new, v_new, ctx_lens, out=None, lse=None, workspace=None,
                             sm_scale=0.0, stream=None):
    """Returns (call, out, lse): call() re-runs the draft attention into out / lse."""
    return _prepare_attn(False, q, k_ctx, v_ctx, k_new, v_new, ctx_lens, None, out, lse, workspace,
                         sm_scale, stream)


def prepare_tree_verify_attn(q, k_ctx, v_ctx, k_new, v_new, ctx_lens, parents, out=None, lse=None,
                             workspace=None, sm_scale=0.0, stream=None):
    """Returns (call, out, lse): call() re-runs the tree-verify attention into out / lse."""
    return _prepare_attn(True, q, k_ctx, v_ctx, k_new, v_new, ctx_lens, parents, out, lse, workspace,
                         sm_scale, stream)


def prepare_greedy_accept(logits, parents, tokens, path_stride=None, outputs=None, workspace=None,
                          stream=None, want_entropy=False):
    """Returns (call, outputs): call() re-runs the acceptance into the outputs dict."""
    args, outputs, ws = _accept_args(logits, parents, tokens, path_stride, outputs, workspace, stream,
                                     want_entropy)
    fn = _accept_fn(want_entropy)
    _check(fn(*args))
    keep = (logits, parents, tokens, outputs, ws)
    return PreparedCall(fn, args, keep), outputs


def prepare_build_tree(draft_logits, roots, budget, first_row=0, horizon=None, outputs=None, workspace=None,
                       stream=None, want_scores=True):
    """Returns (call, outputs): call() re-runs the tree builder into the outputs dict."""
    args, outputs, ws = _tree_args(draft_logits, roots, budget, first_row, horizon, outputs, workspace, stream,
                                   want_scores)
    _check(lib().glance_build_tree(*args))
    keep = (draft_logits, roots, outputs, ws)
    return PreparedCall(lib().glance_build_tree, args, keep), outputs
