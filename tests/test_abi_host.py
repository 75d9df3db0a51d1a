"""C-ABI boundary checks that need no GPU: the library loads, exports every
symbol include/glance.h declares, and rejects bad arguments on the host before
any HIP call.  Every call made here fails validation (at least one argument is
invalid), so no kernel is ever launched with the placeholder pointers used."""

import ctypes
import os
import re

import numpy as np
import pytest

import paper_2609_00355_amd as G

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "glance.h")

FAKE = ctypes.c_void_p(0x10000)   # aligned placeholder; never dereferenced (validation fails first)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(G.LIB_PATH):
        from paper_2609_00355_amd import build
        build.build()
    return G.lib()


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(glance_[a-z_0-9]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(lib):
    names = _declared_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), f"{n} declared in glance.h but not exported"


def test_version_and_status_strings(lib):
    assert G.glance_version() >= 100
    for code in (0, -1, -2, -3, -4):
        assert G.glance_status_string(code)
    assert G.glance_status_string(7) == "unknown status"


def _shape(**kw):
    base = dict(batch=1, n_new=16, n_q_heads=28, n_kv_heads=4, head_dim=128, ctx_capacity=2048,
                dtype=G.GLANCE_BF16)
    base.update(kw)
    return G.attn_shape(**base)


@pytest.mark.parametrize("kw,code", [
    (dict(batch=0), G.GLANCE_ERR_INVALID_ARG),
    (dict(n_new=0), G.GLANCE_ERR_UNSUPPORTED),
    (dict(n_new=65), G.GLANCE_ERR_UNSUPPORTED),
    (dict(n_q_heads=27), G.GLANCE_ERR_INVALID_ARG),
    (dict(n_q_heads=68, n_kv_heads=4), G.GLANCE_ERR_UNSUPPORTED),
    (dict(head_dim=96), G.GLANCE_ERR_UNSUPPORTED),
    (dict(ctx_capacity=-1), G.GLANCE_ERR_INVALID_ARG),
    (dict(dtype=5), G.GLANCE_ERR_UNSUPPORTED),
])
def test_bad_shapes_are_rejected(lib, kw, code):
    s = _shape(**kw)
    assert G.glance_attn_workspace_size(s) == 0
    st = lib.glance_block_draft_attn(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None,
                                     None, 0, None)
    assert st == code, G.glance_last_error()
    assert G.glance_last_error()


def test_null_and_misaligned_pointers(lib):
    s = _shape()
    ws = G.glance_attn_workspace_size(s)
    assert ws > 0
    st = lib.glance_block_draft_attn(ctypes.byref(s), None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None,
                                     FAKE, ws, None)
    assert st == G.GLANCE_ERR_INVALID_ARG and "q" in G.glance_last_error()
    st = lib.glance_block_draft_attn(ctypes.byref(s), ctypes.c_void_p(0x10008), FAKE, FAKE, FAKE, FAKE,
                                     FAKE, FAKE, None, FAKE, ws, None)
    assert st == G.GLANCE_ERR_INVALID_ARG and "aligned" in G.glance_last_error()
    st = lib.glance_tree_verify_attn(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE,
                                     None, FAKE, ws, None)
    assert st == G.GLANCE_ERR_INVALID_ARG and "parents" in G.glance_last_error()


def test_workspace_checks(lib):
    s = _shape()
    ws = G.glance_attn_workspace_size(s)
    st = lib.glance_block_draft_attn(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None,
                                     None, ws, None)
    assert st == G.GLANCE_ERR_WORKSPACE
    st = lib.glance_block_draft_attn(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None,
                                     FAKE, ws - 1, None)
    assert st == G.GLANCE_ERR_WORKSPACE and "too small" in G.glance_last_error()
    st = lib.glance_block_draft_attn(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None,
                                     ctypes.c_void_p(0x10010), ws, None)
    assert st == G.GLANCE_ERR_WORKSPACE and "256" in G.glance_last_error()


def test_workspace_size_depends_on_the_shape_only(lib):
    s = _shape(batch=4, n_new=64, ctx_capacity=16384)
    a = G.glance_attn_workspace_size(s, 1)
    assert a == G.glance_attn_workspace_size(s, 0) > 0
    # 256 workgroups' partials: 32 piece slots x 4 KV heads x 2 row groups,
    # each 224 rows x head_dim fp16 values and a (max, sum) pair of floats
    assert a >= 256 * 224 * (128 * 2 + 8)
    # no hidden inputs: the same size in a child process with a changed environment
    import subprocess
    import sys
    env = dict(os.environ, GLANCE_TARGET_WGS="64", GLANCE_TILES_PER_WAVE="1", GLANCE_ACCEPT_WGS="7")
    code = ("import paper_2609_00355_amd as G; s = G.attn_shape(4, 64, 28, 4, 128, 16384, G.GLANCE_BF16); "
            "print(G.glance_attn_workspace_size(s, 1), G.glance_accept_workspace_size(4, 64, 152064))")
    out = subprocess.run([sys.executable, "-c", code], env=env, cwd=ROOT, capture_output=True, text=True, check=True)
    assert out.stdout.split() == [str(a), str(G.glance_accept_workspace_size(4, 64, 152064))]
    # more sequences than piece slots: one slot per sequence
    big = G.glance_attn_workspace_size(_shape(batch=100, n_new=64, ctx_capacity=128), 1)
    assert big >= 100 * 4 * 2 * 224 * (128 * 2 + 8)


def test_accept_argument_checks(lib):
    assert G.glance_accept_workspace_size(4, 64, 152064) > 0
    assert G.glance_accept_workspace_size(0, 64, 10) == 0
    assert G.glance_accept_workspace_size(1, 65, 10) == 0
    st = lib.glance_greedy_accept(1, 65, 100, G.GLANCE_BF16, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 16, FAKE,
                                  FAKE, 1 << 20, None)
    assert st == G.GLANCE_ERR_UNSUPPORTED
    st = lib.glance_greedy_accept(1, 8, 100, G.GLANCE_BF16, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0, FAKE,
                                  FAKE, 1 << 20, None)
    assert st == G.GLANCE_ERR_INVALID_ARG and "path_stride" in G.glance_last_error()
    st = lib.glance_greedy_accept(1, 8, 100, G.GLANCE_BF16, FAKE, None, FAKE, FAKE, FAKE, FAKE, 8, FAKE,
                                  FAKE, 1 << 20, None)
    assert st == G.GLANCE_ERR_INVALID_ARG and "parents" in G.glance_last_error()
    st = lib.glance_greedy_accept(1, 8, 100, G.GLANCE_BF16, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 8, FAKE,
                                  FAKE, 1, None)
    assert st == G.GLANCE_ERR_WORKSPACE
    # the entropy variant takes the same checks and needs its output pointer
    st = lib.glance_greedy_accept_entropy(1, 8, 100, G.GLANCE_BF16, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 8, FAKE,
                                          None, FAKE, 1 << 20, None)
    assert st == G.GLANCE_ERR_INVALID_ARG and "root_entropy" in G.glance_last_error()
    st = lib.glance_greedy_accept_entropy(1, 65, 100, G.GLANCE_BF16, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 16, FAKE,
                                          FAKE, FAKE, 1 << 20, None)
    assert st == G.GLANCE_ERR_UNSUPPORTED


def _sample(lib, n=8, temperature=1.0, parents=FAKE, draws=FAKE, ws=FAKE, ws_bytes=1 << 20, dtype=G.GLANCE_BF16,
            counter=None):
    return lib.glance_sample_accept(1, n, 100, dtype, FAKE, parents, FAKE, temperature, 2 ** 64 - 1, 2 ** 32 - 1,
                                    counter, draws, FAKE, FAKE, 8, FAKE, ws, ws_bytes, None)


def test_sample_argument_checks(lib):
    for t in (0.0, -1.0, float("inf"), float("nan"), 1e-39):
        assert _sample(lib, temperature=t) == G.GLANCE_ERR_INVALID_ARG
        assert "temperature" in G.glance_last_error()
    assert _sample(lib, n=65) == G.GLANCE_ERR_UNSUPPORTED
    assert _sample(lib, parents=None) == G.GLANCE_ERR_INVALID_ARG and "parents" in G.glance_last_error()
    assert _sample(lib, draws=None) == G.GLANCE_ERR_INVALID_ARG and "draws_out" in G.glance_last_error()
    assert _sample(lib, ws_bytes=1) == G.GLANCE_ERR_WORKSPACE
    assert _sample(lib, ws=ctypes.c_void_p(0x10010)) == G.GLANCE_ERR_WORKSPACE
    assert _sample(lib, dtype=7) == G.GLANCE_ERR_UNSUPPORTED
    assert _sample(lib, counter=ctypes.c_void_p(0x10002)) == G.GLANCE_ERR_INVALID_ARG
    assert "round_counter" in G.glance_last_error()


def _build_tree(lib, batch=1, horizon=15, vocab=152064, budget=63, dtype=G.GLANCE_BF16, logits=FAKE,
                stride=None, roots=FAKE, parents=FAKE, tokens=FAKE, scores=FAKE, ws=FAKE, ws_bytes=1 << 30):
    stride = horizon * vocab if stride is None else stride
    return lib.glance_build_tree(batch, horizon, vocab, budget, dtype, logits, stride, roots, parents, tokens,
                                 scores, ws, ws_bytes, None)


def test_tree_builder_workspace_size(lib):
    a = G.glance_tree_workspace_size(4, 15, 152064, 63)
    assert a > 0
    # candidate lists dominate: rows x 2048 slots x 8 bytes
    assert a >= 4 * 15 * 2048 * 8
    assert G.glance_tree_workspace_size(8, 15, 152064, 63) > a
    assert G.glance_tree_workspace_size(1, 15, 152064, 64) == 0
    assert G.glance_tree_workspace_size(1, 16, 152064, 63) == 0
    assert G.glance_tree_workspace_size(1, 2, 2, 7) == 0          # 2 + 4 strings < 7
    assert G.glance_tree_workspace_size(1, 2, 2, 6) > 0


@pytest.mark.parametrize("kw,code,word", [
    (dict(batch=0), G.GLANCE_ERR_INVALID_ARG, "batch"),
    (dict(horizon=0), G.GLANCE_ERR_INVALID_ARG, "horizon"),
    (dict(horizon=16), G.GLANCE_ERR_UNSUPPORTED, "horizon"),
    (dict(budget=0), G.GLANCE_ERR_INVALID_ARG, "budget"),
    (dict(budget=64), G.GLANCE_ERR_UNSUPPORTED, "budget"),
    (dict(vocab=3, horizon=3, budget=63), G.GLANCE_ERR_INVALID_ARG, "strings"),    # 3 + 9 + 27 < 63
    (dict(vocab=0), G.GLANCE_ERR_INVALID_ARG, "vocab"),
    (dict(dtype=5), G.GLANCE_ERR_UNSUPPORTED, "dtype"),
    (dict(stride=15 * 152064 - 1), G.GLANCE_ERR_INVALID_ARG, "seq_stride"),
    (dict(logits=None), G.GLANCE_ERR_INVALID_ARG, "draft_logits"),
    (dict(logits=ctypes.c_void_p(0x10001)), G.GLANCE_ERR_INVALID_ARG, "aligned"),
    (dict(roots=None), G.GLANCE_ERR_INVALID_ARG, "roots"),
    (dict(parents=None), G.GLANCE_ERR_INVALID_ARG, "parents"),
    (dict(tokens=ctypes.c_void_p(0x10002)), G.GLANCE_ERR_INVALID_ARG, "tokens"),
    (dict(scores=ctypes.c_void_p(0x10002)), G.GLANCE_ERR_INVALID_ARG, "scores"),
    (dict(ws=None), G.GLANCE_ERR_WORKSPACE, "workspace"),
    (dict(ws=ctypes.c_void_p(0x10010)), G.GLANCE_ERR_WORKSPACE, "aligned"),
    (dict(ws_bytes=1024), G.GLANCE_ERR_WORKSPACE, "too small"),
])
def test_tree_builder_argument_checks(lib, kw, code, word):
    assert _build_tree(lib, **kw) == code
    assert word in G.glance_last_error()


def _commit(lib, batch=1, n=64, hkv=4, d=128, cap=4096, dtype=G.GLANCE_BF16, k_new=FAKE, v_new=FAKE,
            alen=FAKE, apath=FAKE, stride=16, k_ctx=FAKE, v_ctx=FAKE, lens=FAKE):
    return lib.glance_commit_path(batch, n, hkv, d, cap, dtype, k_new, v_new, alen, apath, stride, k_ctx, v_ctx,
                                  lens, None)


@pytest.mark.parametrize("kw,code,word", [
    (dict(batch=0), G.GLANCE_ERR_INVALID_ARG, "batch"),
    (dict(n=0), G.GLANCE_ERR_UNSUPPORTED, "n_nodes"),
    (dict(n=65), G.GLANCE_ERR_UNSUPPORTED, "n_nodes"),
    (dict(hkv=0), G.GLANCE_ERR_INVALID_ARG, "n_kv_heads"),
    (dict(d=0), G.GLANCE_ERR_UNSUPPORTED, "head_dim"),
    (dict(d=2048), G.GLANCE_ERR_UNSUPPORTED, "head_dim"),
    (dict(cap=0), G.GLANCE_ERR_INVALID_ARG, "ctx_capacity"),
    (dict(stride=0), G.GLANCE_ERR_INVALID_ARG, "path_stride"),
    (dict(dtype=7), G.GLANCE_ERR_UNSUPPORTED, "dtype"),
    (dict(k_new=None), G.GLANCE_ERR_INVALID_ARG, "k_new"),
    (dict(v_ctx=None), G.GLANCE_ERR_INVALID_ARG, "v_ctx"),
    (dict(lens=None), G.GLANCE_ERR_INVALID_ARG, "ctx_lens"),
    (dict(k_ctx=ctypes.c_void_p(0x10001)), G.GLANCE_ERR_INVALID_ARG, "aligned"),
    (dict(apath=ctypes.c_void_p(0x10002)), G.GLANCE_ERR_INVALID_ARG, "accept_path"),
])
def test_commit_argument_checks(lib, kw, code, word):
    assert _commit(lib, **kw) == code
    assert word in G.glance_last_error()


@pytest.mark.parametrize("parents,tokens,max_depth,ok", [
    ([-1], None, 15, True),
    ([-1, 0, 0, 1, 3], [9, 1, 2, 3, 4], 15, True),
    ([0, 0], None, 15, False),                 # root must have parent -1
    ([-1, 1], None, 15, False),                # parent must precede the child
    ([-1, 0, 3, 0], None, 15, False),
    ([-1, 0, 1, 2, 3], None, 3, False),        # depth 4 > 3
    ([-1, 0, 0], [5, 7, 7], 15, False),        # siblings repeat a token
    ([-1, 0, 1], [5, 7, 7], 15, True),         # same token at different depths is fine
])
def test_validate_tree(lib, parents, tokens, max_depth, ok):
    good, msg = G.glance_validate_tree(parents, tokens, max_depth)
    assert good == ok, msg
    if not ok:
        assert msg


def test_validate_generated_trees(lib):
    from workloads import configs
    w = configs.WORKLOADS["verify_4k"]
    par, tok = configs.tree_inputs(w, seed=3)
    good, msg = G.glance_validate_tree(par[0].numpy(), tok[0].numpy(), 15)
    assert good, msg


def test_kernel_events_need_both_or_neither(lib):
    assert lib.glance_set_kernel_events(FAKE, None) == G.GLANCE_ERR_INVALID_ARG
    assert lib.glance_set_kernel_events(None, None) == G.GLANCE_OK


# The C contract of the hot path's boundary: return type and parameter types,
# in order, of each call, and the layout of the shape struct and the enums.
BOUNDARY = {
    "glance_block_draft_attn": ("glance_status", [
        "const glance_attn_shape*", "const void*", "const void*", "const void*", "const void*", "const void*",
        "const int32_t*", "void*", "float*", "void*", "size_t", "hipStream_t"]),
    "glance_tree_verify_attn": ("glance_status", [
        "const glance_attn_shape*", "const void*", "const void*", "const void*", "const void*", "const void*",
        "const int32_t*", "const int32_t*", "void*", "float*", "void*", "size_t", "hipStream_t"]),
    "glance_greedy_accept": ("glance_status", [
        "int32_t", "int32_t", "int32_t", "glance_dtype", "const void*", "const int32_t*", "const int32_t*",
        "int32_t*", "int32_t*", "int32_t*", "int32_t", "int32_t*", "void*", "size_t", "hipStream_t"]),
    "glance_attn_workspace_size": ("size_t", ["const glance_attn_shape*", "int"]),
    "glance_accept_workspace_size": ("size_t", ["int32_t", "int32_t", "int32_t"]),
    "glance_validate_tree": ("glance_status", ["int32_t", "const int32_t*", "const int32_t*", "int32_t"]),
    "glance_status_string": ("const char*", ["glance_status"]),
    "glance_last_error": ("const char*", []),
}


def _prototypes():
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    text = re.sub(r"\s+", " ", text)
    protos = {}
    for m in re.finditer(r"([A-Za-z_][A-Za-z_0-9 ]*?\*?) ?\b(glance_[a-z_0-9]+) ?\(([^()]*)\) ?;", text):
        ret, name, params = m.group(1).strip(), m.group(2), m.group(3).strip()
        types = []
        if params and params != "void":
            for prm in params.split(","):
                prm = prm.strip().replace(" *", "*")
                words = prm.replace("*", "* ").split()
                # the last word is the parameter's name
                types.append(" ".join(words[:-1]).replace("* ", "*").replace(" *", "*").strip())
        protos[name] = (ret.replace(" *", "*"), types)
    return protos


@pytest.mark.parametrize("name", sorted(BOUNDARY))
def test_boundary_prototype(name):
    protos = _prototypes()
    assert name in protos, f"{name} is not declared in glance.h"
    assert protos[name] == BOUNDARY[name]


def test_boundary_types():
    text = re.sub(r"\s+", " ", re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S))
    fields = re.search(r"typedef struct \{(.*?)\} glance_attn_shape;", text).group(1)
    assert [f.split()[-1] for f in fields.split(";") if f.strip()] == [
        "batch", "n_new", "n_q_heads", "n_kv_heads", "head_dim", "ctx_capacity", "sm_scale", "dtype"]
    assert [f.split()[0] for f in fields.split(";") if f.strip()] == ["int32_t"] * 6 + ["float", "glance_dtype"]
    assert ctypes.sizeof(G.AttnShape) == 32
    assert (G.GLANCE_OK, G.GLANCE_ERR_INVALID_ARG, G.GLANCE_ERR_UNSUPPORTED, G.GLANCE_ERR_WORKSPACE,
            G.GLANCE_ERR_HIP) == (0, -1, -2, -3, -4)
    assert (G.GLANCE_F32, G.GLANCE_BF16) == (0, 1)
    assert re.search(r"GLANCE_OK = 0, GLANCE_ERR_INVALID_ARG = -1, GLANCE_ERR_UNSUPPORTED = -2, "
                     r"GLANCE_ERR_WORKSPACE = -3, GLANCE_ERR_HIP = -4 \} glance_status;", text)
    assert re.search(r"typedef enum \{ GLANCE_F32 = 0, GLANCE_BF16 = 1 \} glance_dtype;", text)


def test_noalloc_accept_host_checks(lib):
    """The allocation-free acceptance rejects, before any HIP call, shapes whose
    scratch would not fit its static buffer, and the usual bad arguments."""
    st = lib.glance_greedy_accept_noalloc(4096, 64, 1000, G.GLANCE_BF16, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 16,
                                          FAKE, None)
    assert st == G.GLANCE_ERR_UNSUPPORTED and "static buffer" in G.glance_last_error()
    st = lib.glance_greedy_accept_noalloc(1, 8, 100, G.GLANCE_BF16, FAKE, None, FAKE, FAKE, FAKE, FAKE, 8, FAKE,
                                          None)
    assert st == G.GLANCE_ERR_INVALID_ARG and "parents" in G.glance_last_error()
    st = lib.glance_greedy_accept_noalloc(1, 65, 100, G.GLANCE_BF16, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 8, FAKE,
                                          None)
    assert st == G.GLANCE_ERR_UNSUPPORTED
