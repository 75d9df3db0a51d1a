"""Bit-exact parity of the HIP greedy acceptance with the oracle: argmax of
every row (lowest index on ties), accepted length, accepted path and the
bonus token, on planted logits, tie fixtures and edge cases; the optional root
entropy within fp32 rounding of the float64 definition."""

import numpy as np
import pytest
import torch

import paper_2609_00355_amd as G
from gpu_helpers import assert_accept_equal, ensure_lib, run_accept
from oracle import accept as OA
from workloads import configs as C

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_lib()


def _round(name, seed=0, batch=None):
    w = C.WORKLOADS[name]
    if batch is not None:
        w = C.custom_workload(name, batch=batch)
    par, tok = C.tree_inputs(w, seed)
    logits = C.planted_logits(w, par, tok, seed)
    return logits, par, tok


@pytest.mark.parametrize("name", ["tiny_fp32", "verify_4k"])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_planted_rounds(name, seed):
    logits, par, tok = _round(name, seed)
    got = run_accept(logits, par, tok, path_stride=16)
    ref = assert_accept_equal(got, logits, par, tok, path_stride=16)
    print(f"[{name} seed {seed}] accept_len={ref['accept_len'].tolist()}", flush=True)


def test_doc_16k_and_ragged_mix_logits():
    for name in ("doc_16k", "ragged_mix"):
        logits, par, tok = _round(name, 0)
        got = run_accept(logits, par, tok, path_stride=16)
        ref = assert_accept_equal(got, logits, par, tok, path_stride=16)
        print(f"[{name}] mean accept_len={ref['accept_len'].mean():.2f}", flush=True)


def _tie_logits(vocab, dtype, ties, batch=1, n=4):
    """Rows of N(0,1) with the maximum value 9.0 planted at every index in ``ties``."""
    g = torch.Generator().manual_seed(1234)
    x = torch.randn((batch, n, vocab), generator=g)
    for b in range(batch):
        for v in range(n):
            for j in ties:
                x[b, v, j] = 9.0
    return x.to(dtype)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("ties", [(0, 152063), (5, 6), (4095, 4096), (70000, 8, 152000), (151999,)])
def test_ties_resolve_to_lowest_index(dtype, ties):
    vocab = 152064
    logits = _tie_logits(vocab, dtype, ties)
    par = torch.tensor([[-1, 0, 0, 1]], dtype=torch.int32)
    tok = torch.tensor([[3, min(ties), max(ties), 11]], dtype=torch.int32)
    got = run_accept(logits, par, tok)
    assert (got["argmax"] == min(ties)).all()
    assert_accept_equal(got, logits, par, tok)


@pytest.mark.parametrize("vocab", [1, 7, 1000, 4097, 152063])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_odd_vocab_sizes(vocab, dtype):
    g = torch.Generator().manual_seed(vocab)
    logits = torch.randn((2, 5, vocab), generator=g).to(dtype)
    par = torch.tensor([[-1, 0, 1, 1, 0], [-1, 0, 0, 2, 3]], dtype=torch.int32)
    am = logits.float().argmax(-1)
    tok = torch.tensor([[0, int(am[0, 0]), int(am[0, 1]), 1, 2],
                        [0, 5, int(am[1, 0]), int(am[1, 2]), int(am[1, 3])]], dtype=torch.int32)
    got = run_accept(logits, par, tok)
    assert_accept_equal(got, logits, par, tok)


def test_signed_zero_and_nan_semantics():
    vocab = 64
    x = torch.full((1, 3, vocab), -1.0)
    x[0, 0, 40] = -0.0
    x[0, 0, 9] = 0.0            # -0 == +0: the lowest index (9) wins
    x[0, 1, 50] = float("nan")
    x[0, 1, 20] = float("nan")  # first NaN wins
    x[0, 1, 3] = 100.0
    x[0, 2, 33] = -float("nan")  # negative-signed NaN still counts as the maximum
    x[0, 2, 2] = float("inf")
    par = torch.tensor([[-1, 0, 1]], dtype=torch.int32)
    tok = torch.tensor([[0, 9, 20]], dtype=torch.int32)
    for dtype in (torch.float32, torch.bfloat16):
        logits = x.to(dtype)
        got = run_accept(logits, par, tok)
        assert got["argmax"].tolist() == [[9, 20, 33]]
        assert_accept_equal(got, logits, par, tok)
        assert got["accept_len"].tolist() == [2]


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_special_values_in_long_rows(dtype):
    """Signed zeros, NaNs, constant rows and a maximum in the last vector of a
    152064-wide row: the vectorised scan must hand every one of these to the
    same answer as the plain definition."""
    vocab = 152064
    g = torch.Generator().manual_seed(77)
    x = torch.full((1, 12, vocab), -2.0)
    x[0, 0, 100000] = -0.0
    x[0, 0, 120000] = 0.0             # -0 ties with the later +0: 100000
    x[0, 1, 90000] = -0.0             # -0 alone is the maximum: 90000
    x[0, 2] = 0.0                     # constant +0: 0
    x[0, 3] = -float("inf")           # constant -inf: 0
    x[0, 4, 151000] = float("nan")
    x[0, 4, 150000] = -float("nan")   # first NaN of either sign: 150000
    x[0, 5] = torch.randn(vocab, generator=g)
    x[0, 5, vocab - 1] = 50.0         # maximum in the row's last element: vocab - 1
    x[0, 6] = 1.5                     # constant: 0
    x[0, 7] = torch.randn(vocab, generator=g)
    x[0, 7, 8007] = 50.0
    x[0, 7, 8008] = 50.0              # tie across a chunk boundary of this 12-row shape: 8007
    x[0, 8] = torch.randn(vocab, generator=g)
    x[0, 8, 16383] = x[0, 8, 16384] = x[0, 8, 40000] = 30.0   # 16383
    x[0, 9] = torch.randn(vocab, generator=g)
    x[0, 9, 130000] = float("inf")
    x[0, 9, 123457] = float("inf")    # first +inf: 123457
    x[0, 10] = -float("inf")
    x[0, 10, 99999] = -5.0            # the one finite value: 99999
    x[0, 11, 5000] = 2e-40
    x[0, 11, 70000] = 3e-40           # subnormal maximum: 70000
    want = [100000, 90000, 0, 0, 150000, vocab - 1, 0, 8007, 16383, 123457, 99999, 70000]
    x = x[:, : len(want)]
    par = torch.arange(-1, len(want) - 1, dtype=torch.int32)[None]
    tok = torch.tensor([want[:1] + want[:-1]], dtype=torch.int32)
    logits = x.to(dtype)
    got = run_accept(logits, par, tok, path_stride=16)
    assert got["argmax"].tolist() == [want]
    assert_accept_equal(got, logits, par, tok, path_stride=16)


@pytest.mark.parametrize("vocab", [8, 2048, 16384, 16392, 32768 + 8, 65536 + 2048])
def test_vector_scan_group_boundaries(vocab):
    """bf16 rows whose lengths sit on and next to the scan's 8-value vector and
    its 16384-value unrolled step, with the maximum planted in the last element and, in a second
    row, ties at the first and last element."""
    g = torch.Generator().manual_seed(vocab)
    x = torch.randn((2, 3, vocab), generator=g)
    x[:, 0, vocab - 1] = 40.0
    x[:, 1, 0] = 40.0
    x[:, 1, vocab - 1] = 40.0
    logits = x.to(torch.bfloat16)
    par = torch.tensor([[-1, 0, 1], [-1, 0, 0]], dtype=torch.int32)
    tok = torch.tensor([[5, vocab - 1, 0], [5, 0, 1]], dtype=torch.int32)
    got = run_accept(logits, par, tok)
    assert got["argmax"][:, :2].tolist() == [[vocab - 1, 0], [vocab - 1, 0]]
    assert_accept_equal(got, logits, par, tok)


def test_path_stride_truncates_but_counts():
    n = 20
    par = torch.arange(-1, n - 1, dtype=torch.int32)[None]
    tok = torch.arange(100, 100 + n, dtype=torch.int32)[None]
    logits = torch.zeros((1, n, 200))
    for v in range(n - 1):
        logits[0, v, 100 + v + 1] = 1.0
    got = run_accept(logits, par, tok, path_stride=5)
    assert got["accept_len"].tolist() == [n - 1]
    assert got["accept_path"].tolist() == [[0, 1, 2, 3, 4]]
    assert got["next_root"].tolist() == [0]


def test_malformed_parents_terminate():
    """Parents that point forward or out of range end the walk instead of looping."""
    par = torch.tensor([[-1, 0, 5, 1, 99, 2]], dtype=torch.int32)
    tok = torch.tensor([[0, 1, 2, 3, 4, 5]], dtype=torch.int32)
    logits = torch.zeros((1, 6, 8))
    for v in range(6):
        logits[0, v, (v + 1) % 8] = 1.0
    got = run_accept(logits, par, tok)
    # row 0 -> token 1 -> node 1; row 1 -> token 2: node 2's parent is 5 (not 1), so stop
    assert got["accept_len"].tolist() == [1]
    assert got["next_root"].tolist() == [2]


def test_many_sequences():
    w = C.custom_workload("tiny_fp32", batch=37)
    par, tok = C.tree_inputs(w, 6)
    logits = C.planted_logits(w, par, tok, 6)
    got = run_accept(logits, par, tok, path_stride=16)
    assert_accept_equal(got, logits, par, tok, path_stride=16)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("case", ["planted", "uniform", "masked", "small_vocab"])
def test_root_entropy(dtype, case):
    """Entropy of each sequence's row 0 (fused into the argmax pass) against float64."""
    w = C.WORKLOADS["verify_4k"]
    batch, n = 3, 8
    par, tok = C.tree_inputs(w, seed=5, batch=batch, n=n)
    vocab = 7 if case == "small_vocab" else w.vocab
    g = torch.Generator().manual_seed(11)
    logits = (torch.randn(batch, n, vocab, generator=g) * 1.4).to(dtype)
    if case == "planted":
        logits[:, 0, 5] = 14.0          # a confident root row
    elif case == "uniform":
        logits[:, 0] = 0.5
    elif case == "masked":
        logits[:, 0, 1000:] = float("-inf")
    tok = tok % vocab
    res = G.glance_greedy_accept(logits.cuda(), par.cuda(), tok.cuda(), want_entropy=True)
    h = res["root_entropy"].cpu().numpy()
    for b in range(batch):
        ref = OA.row_entropy(logits[b, 0])
        assert abs(h[b] - ref) <= 2e-4 + 2e-5 * abs(ref), (b, h[b], ref)
    if case == "uniform":
        assert abs(h[0] - np.log(vocab)) < 2e-4 + 2e-5 * np.log(vocab)
    # the argmax and walk are unchanged by the extra output
    plain = G.glance_greedy_accept(logits.cuda(), par.cuda(), tok.cuda())
    for k in ("argmax", "accept_len", "accept_path", "next_root"):
        assert torch.equal(plain[k], res[k])


def test_one_workspace_across_calls_and_shapes():
    """One workspace serves greedy and sampling calls of different shapes in
    turn: nothing a call reads from it was left by an earlier call."""
    shapes = [(4, 64, 152064), (1, 16, 1000), (6, 33, 50000), (4, 64, 152064)]
    need = max(G.glance_accept_workspace_size(*s) for s in shapes)
    ws = torch.full((need,), 0xA5, dtype=torch.uint8, device="cuda")  # stale bytes
    for i, (batch, n, vocab) in enumerate(shapes):
        w = C.custom_workload("verify_4k", batch=batch, n_tree=n, depth_cap=min(15, n - 1), vocab=vocab)
        par, tok = C.tree_inputs(w, 20 + i)
        logits = C.planted_logits(w, par, tok, 20 + i)
        got = G.glance_greedy_accept(logits.cuda(), par.cuda(), tok.cuda(), path_stride=16, workspace=ws)
        torch.cuda.synchronize()
        assert_accept_equal({k: v.cpu().numpy() for k, v in got.items()}, logits, par, tok, path_stride=16)
        smp = G.glance_sample_accept(logits.cuda(), par.cuda(), tok.cuda(), 1.0, 5, i, path_stride=16,
                                     workspace=ws)
        torch.cuda.synchronize()
        assert int(smp["accept_len"].min()) >= 0
        print(f"[workspace reuse] call {i}: batch {batch} n {n} vocab {vocab} ok", flush=True)
