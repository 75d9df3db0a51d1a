"""Bit-exact parity of the HIP sampling walk with the oracle: every row's
Gumbel-max draw (Philox4x32-10 noise, the fixed fp32 logarithm), the accepted
length and path and the next root, over temperatures, seeds, rounds, dtypes,
vocabulary sizes and special values; at the full doc_16k shape on sampled rows
plus the walk recomputed from the GPU's own draws."""

import numpy as np
import pytest
import torch

import paper_2609_00355_amd as G
from gpu_helpers import ensure_lib
from oracle import accept as OA
from oracle import sampling as S
from workloads import configs as C

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_lib()


def _run(logits, par, tok, temperature, seed, round_, path_stride=16):
    res = G.glance_sample_accept(logits.cuda(), par.cuda(), tok.cuda(), temperature, seed, round_,
                                 path_stride=path_stride)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in res.items()}


def _check(got, logits, par, tok, temperature, seed, round_, path_stride=16, rows=None):
    """Draws of the given rows (all by default) and, when all rows are checked,
    the walk; the walk is always recomputed from the GPU's own draws."""
    batch, n, _ = logits.shape
    par_np, tok_np = par.numpy(), tok.numpy()
    for b in range(batch):
        for v in (range(n) if rows is None else rows):
            want = S.sample_row(logits[b, v], temperature, seed, round_, b, v)
            assert got["draws"][b, v] == want, (b, v, got["draws"][b, v], want)
        a, path, nr = OA.greedy_walk(got["draws"][b].tolist(), par_np[b].tolist(), tok_np[b].tolist())
        assert got["accept_len"][b] == a, (b, got["accept_len"][b], a)
        want_path = (list(path) + [-1] * path_stride)[:path_stride]
        assert got["accept_path"][b].tolist() == want_path
        assert got["next_root"][b] == nr


def _peaked(batch, n, vocab, seed, dtype, peak=15.0, sigma=1.0):
    """N(0, sigma^2) rows with every child's token raised to `peak` in its
    parent's row, so that at T = 1 the draws mostly follow the tree."""
    w = C.custom_workload("verify_4k", vocab=vocab)
    par, tok = C.tree_inputs(w, seed=seed, batch=batch, n=n)
    tok = tok % vocab
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((batch, n, vocab), generator=g) * sigma
    for b in range(batch):
        for c in range(1, n):
            x[b, int(par[b, c]), int(tok[b, c])] = peak
    return x.to(dtype), torch.as_tensor(par), torch.as_tensor(tok)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("temperature", [1.0, 0.5, 0.7, 2.0])
def test_draws_and_walk_match_oracle(dtype, temperature):
    logits, par, tok = _peaked(2, 16, 4097, seed=3, dtype=dtype)
    for seed, round_ in [(0, 0), (12345, 7), (2 ** 64 - 1, 2 ** 32 - 1)]:
        got = _run(logits, par, tok, temperature, seed, round_)
        _check(got, logits, par, tok, temperature, seed, round_)
    print(f"[{dtype} T={temperature}] accept_len={got['accept_len'].tolist()}", flush=True)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_full_vocab_rows(dtype):
    """152064-wide rows (the target's vocabulary): several chunks per row and a
    deep accepted path."""
    logits, par, tok = _peaked(1, 64, 152064, seed=8, dtype=dtype)
    got = _run(logits, par, tok, 1.0, seed=99, round_=4)
    _check(got, logits, par, tok, 1.0, 99, 4)
    assert got["accept_len"][0] >= 3
    print(f"[{dtype}] accept_len={got['accept_len'].tolist()}", flush=True)


@pytest.mark.parametrize("vocab", [1, 2, 3, 7, 8, 1000, 1024, 1025, 4096 + 5])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_odd_vocab_sizes(vocab, dtype):
    g = torch.Generator().manual_seed(vocab)
    logits = torch.randn((2, 5, vocab), generator=g).to(dtype)
    par = torch.tensor([[-1, 0, 1, 1, 0], [-1, 0, 0, 2, 3]], dtype=torch.int32)
    tok = torch.tensor([[0, 1, 2, 3, 4], [0, 5, 6, 7, 8]], dtype=torch.int32) % vocab
    for seed in (1, 2, 3):
        got = _run(logits, par, tok, 1.0, seed, 0)
        _check(got, logits, par, tok, 1.0, seed, 0)


def test_unaligned_rows_take_the_scalar_loads():
    """A logits view that starts 4 bytes into its buffer and odd row lengths:
    the four-token vector loads must switch off and the answer stay exact."""
    g = torch.Generator().manual_seed(5)
    base = torch.randn((2 * 6 * 1001 + 1,), generator=g)
    logits = base[1:].view(2, 6, 1001)
    par = torch.tensor([[-1, 0, 1, 2, 3, 4]] * 2, dtype=torch.int32)
    tok = torch.tensor([[0, 1, 2, 3, 4, 5]] * 2, dtype=torch.int32)
    res = G.glance_sample_accept(base.cuda()[1:].view(2, 6, 1001), par.cuda(), tok.cuda(), 1.0, 17, 3,
                                 path_stride=16)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in res.items()}
    _check(got, logits, par, tok, 1.0, 17, 3)


def test_constant_and_masked_rows():
    """Rows where the noise alone decides (constant logits), rows with most
    tokens masked to -inf, an all -inf row (draw 0: every value ties), and a
    row with one finite token."""
    vocab = 5000
    x = torch.zeros((1, 6, vocab))
    x[0, 1] = float("-inf")
    x[0, 1, 100:140] = 0.25
    x[0, 2] = float("-inf")
    x[0, 3] = float("-inf")
    x[0, 3, 4321] = -80.0
    x[0, 4] = 3.0
    x[0, 5, ::2] = float("-inf")
    par = torch.tensor([[-1, 0, 1, 2, 3, 4]], dtype=torch.int32)
    tok = torch.tensor([[0, 1, 2, 3, 4, 5]], dtype=torch.int32)
    for dtype in (torch.float32, torch.bfloat16):
        logits = x.to(dtype)
        for seed in range(4):
            got = _run(logits, par, tok, 1.0, seed, 1)
            _check(got, logits, par, tok, 1.0, seed, 1)
            assert 100 <= got["draws"][0, 1] < 140
            assert got["draws"][0, 2] == 0
            assert got["draws"][0, 3] == 4321
            assert got["draws"][0, 5] % 2 == 1


def test_nan_and_inf():
    vocab = 3000
    x = torch.randn((1, 4, vocab), generator=torch.Generator().manual_seed(2))
    x[0, 0, 2500] = float("nan")
    x[0, 0, 1700] = float("nan")      # first NaN wins
    x[0, 1, 10] = float("inf")
    x[0, 1, 20] = float("inf")        # +inf + noise ties at +inf: lowest index
    x[0, 2, 5] = float("-nan")
    x[0, 3, 2999] = 3.0e38            # huge finite values next to their overflow under 1/T
    x[0, 3, 7] = -3.0e38
    par = torch.tensor([[-1, 0, 1, 2]], dtype=torch.int32)
    tok = torch.tensor([[0, 1700, 10, 5]], dtype=torch.int32)
    for dtype in (torch.float32, torch.bfloat16):
        for temperature in (1.0, 0.5):
            logits = x.to(dtype)
            got = _run(logits, par, tok, temperature, 3, 0)
            _check(got, logits, par, tok, temperature, 3, 0)
            assert got["draws"][0, :4].tolist()[:3] == [1700, 10, 5]


@pytest.mark.parametrize("temperature", [0.01, 0.001, 30.0])
def test_extreme_temperatures(temperature):
    """Small T spreads z / T far beyond the noise range (most tokens are skipped
    by the bound, the rest must still be exact); large T flattens the rows so
    the noise dominates."""
    g = torch.Generator().manual_seed(int(temperature * 1000))
    logits = torch.randn((2, 8, 20000), generator=g)
    logits[:, :, 123] += 0.002        # a near tie with the row maximum region
    par = torch.tensor([[-1, 0, 1, 2, 3, 4, 5, 6]] * 2, dtype=torch.int32)
    tok = torch.tensor([[0, 1, 2, 3, 4, 5, 6, 7]] * 2, dtype=torch.int32)
    for seed in (5, 6):
        got = _run(logits, par, tok, temperature, seed, 2)
        _check(got, logits, par, tok, temperature, seed, 2)


def test_near_ties_at_the_filter_margin():
    """Rows of two logit levels 24 ln 2 apart and levels within a few ulp of
    each other: the candidate filter's bound and slack are tested where they
    are tight (a wrong skip changes a draw)."""
    vocab = 65536
    g = torch.Generator().manual_seed(9)
    x = torch.zeros((1, 8, vocab))
    x[0, 0] = torch.where(torch.rand(vocab, generator=g) < 0.001, 24 * np.log(2.0), 0.0)
    x[0, 1] = torch.where(torch.rand(vocab, generator=g) < 0.5, 16.0, 16.0 - 2 ** -19)
    x[0, 2] = torch.randn(vocab, generator=g) * 1e-6 + 5.0
    x[0, 3] = torch.where(torch.rand(vocab, generator=g) < 0.01, 17.0, 0.0)
    x[0, 4] = torch.arange(vocab, dtype=torch.float32) * (20.0 / vocab)
    x[0, 5] = -torch.arange(vocab, dtype=torch.float32) * (20.0 / vocab)
    x[0, 6] = torch.randn(vocab, generator=g) * 8
    x[0, 7] = torch.randn(vocab, generator=g) * 0.01
    par = torch.arange(-1, 7, dtype=torch.int32)[None]
    tok = torch.arange(0, 8, dtype=torch.int32)[None]
    for seed in range(6):
        got = _run(x, par, tok, 1.0, seed, seed)
        _check(got, x, par, tok, 1.0, seed, seed)


def test_many_sequences_and_rounds_differ():
    logits, par, tok = _peaked(9, 24, 2000, seed=4, dtype=torch.bfloat16, peak=3.0)
    a = _run(logits, par, tok, 1.0, 77, 0)
    _check(a, logits, par, tok, 1.0, 77, 0)
    b = _run(logits, par, tok, 1.0, 77, 1)
    _check(b, logits, par, tok, 1.0, 77, 1)
    assert (a["draws"] != b["draws"]).mean() > 0.5


def test_doc_16k_full_shape_sampled_rows():
    """The bench's shape (4 sequences x 64 rows x 152064, bf16): sampled rows
    against the oracle, the walk recomputed from all GPU draws."""
    w = C.WORKLOADS["doc_16k"]
    par, tok = C.tree_inputs(w, 0)
    logits = torch.as_tensor(C.planted_logits(w, par, tok, 0))
    par, tok = torch.as_tensor(par), torch.as_tensor(tok)
    got = _run(logits, par, tok, 1.0, 2026, 11)
    _check(got, logits, par, tok, 1.0, 2026, 11, rows=[0, 1, 17, 40, 63])


def test_host_checks():
    logits = torch.zeros((1, 2, 10), device="cuda")
    par = torch.tensor([[-1, 0]], dtype=torch.int32, device="cuda")
    tok = torch.tensor([[0, 1]], dtype=torch.int32, device="cuda")
    for bad in (0.0, -1.0, float("inf"), float("nan"), 1e-40):
        with pytest.raises(G.GlanceError):
            G.glance_sample_accept(logits, par, tok, bad, 0, 0)
    with pytest.raises(ValueError):
        G.glance_sample_accept(logits, par, tok, 1.0, -1, 0)


def test_device_round_counter_gives_fresh_noise_on_graph_replays():
    """With a device round counter the round used is round_ + counter and the
    call advances the counter: eager calls and the replays of a captured HIP
    graph each draw the next round's noise (checked against the oracle at
    that round), with the program's own synchronisation between replays."""
    logits, par, tok = _peaked(2, 8, 3000, seed=12, dtype=torch.bfloat16, peak=3.0)
    dl, dp, dt = logits.cuda(), par.cuda(), tok.cuda()
    base, seed = 100, 5
    counter = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.zeros(G.glance_accept_workspace_size(2, 8, 3000), dtype=torch.uint8, device="cuda")
    out = G.glance_sample_accept(dl, dp, dt, 1.0, seed, base, path_stride=16, workspace=ws, round_counter=counter)
    torch.cuda.synchronize()
    assert int(counter.item()) == 1
    _check({k: v.cpu().numpy() for k, v in out.items()}, logits, par, tok, 1.0, seed, base)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        G.glance_sample_accept(dl, dp, dt, 1.0, seed, base, path_stride=16, outputs=out, workspace=ws,
                               round_counter=counter)
    torch.cuda.synchronize()
    assert int(counter.item()) == 1                          # capture records, it does not run
    seen = []
    for r in range(1, 5):
        g.replay()
        torch.cuda.synchronize()
        got = {k: v.cpu().numpy() for k, v in out.items()}
        _check(got, logits, par, tok, 1.0, seed, base + r)
        assert int(counter.item()) == r + 1
        seen.append(got["draws"].copy())
    assert any((a != b).any() for a, b in zip(seen, seen[1:]))
    # without a counter the same by-value round gives the same draws
    a = _run(logits, par, tok, 1.0, seed, base + 3)
    assert np.array_equal(a["draws"], seen[2])


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_root_only_trees(dtype):
    """n_nodes = 1 (the tree is just the root): nothing is accepted and the
    next root is the root row's draw (sampling) or argmax (greedy)."""
    g = torch.Generator().manual_seed(31)
    logits = torch.randn((3, 1, 5000), generator=g).to(dtype)
    par = torch.full((3, 1), -1, dtype=torch.int32)
    tok = torch.tensor([[7], [8], [9]], dtype=torch.int32)
    got = _run(logits, par, tok, 0.8, 99, 5, path_stride=1)
    _check(got, logits, par, tok, 0.8, 99, 5, path_stride=1)
    assert got["accept_len"].tolist() == [0, 0, 0]
    assert got["next_root"].tolist() == got["draws"][:, 0].tolist()
    greedy = G.glance_greedy_accept(logits.cuda(), par.cuda(), tok.cuda(), path_stride=1)
    torch.cuda.synchronize()
    assert greedy["accept_len"].cpu().tolist() == [0, 0, 0]
    assert greedy["next_root"].cpu().tolist() == logits.float().argmax(-1)[:, 0].tolist()
    assert greedy["accept_path"].cpu().tolist() == [[0], [0], [0]]
