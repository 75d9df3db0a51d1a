"""GPU parity of the commit (glance_commit_path) against the oracle
(oracle/commit.py): the caches and lengths after the commit must equal the
oracle's bit for bit (a copy involves no arithmetic)."""

import numpy as np
import pytest
import torch

import paper_2609_00355_amd as G
from oracle import accept as OA
from oracle import commit as OC
from workloads import configs as W
from workloads import trees as WT

from gpu_helpers import ensure_lib

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_lib()


def _random_case(seed, batch, n, hkv, d, cap, dtype, stride=16, ctx=None):
    g = torch.Generator().manual_seed(seed)
    k_ctx = torch.randn(batch, hkv, cap, d, generator=g).to(dtype)
    v_ctx = torch.randn(batch, hkv, cap, d, generator=g).to(dtype)
    k_new = torch.randn(batch, n, hkv, d, generator=g).to(dtype)
    v_new = torch.randn(batch, n, hkv, d, generator=g).to(dtype)
    rng = np.random.default_rng(seed)
    ctx = rng.integers(0, cap - 16, size=batch) if ctx is None else np.asarray(ctx)
    alen = np.zeros(batch, dtype=np.int32)
    apath = np.full((batch, stride), -1, dtype=np.int32)
    for b in range(batch):
        par, _ = WT.best_first_tree(n, 15, (1, 2, 4), 100, (seed, b))
        leaf = int(rng.integers(0, n))
        chain = [leaf]
        while chain[-1] != 0:
            chain.append(int(par[chain[-1]]))
        chain = chain[::-1]
        alen[b] = len(chain) - 1
        apath[b, :min(len(chain), stride)] = chain[:stride]
    return dict(k_ctx=k_ctx, v_ctx=v_ctx, k_new=k_new, v_new=v_new,
                ctx=torch.as_tensor(ctx.astype(np.int32)), alen=torch.as_tensor(alen),
                apath=torch.as_tensor(apath))


def _to_bits(t):
    t = torch.as_tensor(t)
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _check(c):
    dev = {k: v.cuda() for k, v in c.items()}
    G.glance_commit_path(dev["k_new"], dev["v_new"], dev["alen"], dev["apath"], dev["k_ctx"], dev["v_ctx"],
                         dev["ctx"])
    torch.cuda.synchronize()
    # oracle on the integer bit patterns (a copy: exact for any dtype)
    kb, vb = _to_bits(c["k_ctx"]).numpy(), _to_bits(c["v_ctx"]).numpy()
    knb, vnb = _to_bits(c["k_new"]).numpy(), _to_bits(c["v_new"]).numpy()
    kc, vc, lens = OC.commit_kv(kb, vb, c["ctx"].numpy(), knb, vnb, c["alen"].numpy(), c["apath"].numpy())
    np.testing.assert_array_equal(dev["ctx"].cpu().numpy(), lens)
    np.testing.assert_array_equal(_to_bits(dev["k_ctx"].cpu()).numpy(), kc)
    np.testing.assert_array_equal(_to_bits(dev["v_ctx"].cpu()).numpy(), vc)
    return lens


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("hkv,d", [(4, 128), (1, 64), (2, 6), (3, 5)])
def test_random_paths(dtype, hkv, d):
    c = _random_case(hkv * 100 + d, batch=4, n=64, hkv=hkv, d=d, cap=200, dtype=dtype)
    _check(c)


def test_root_only_and_full_chain():
    c = _random_case(7, batch=2, n=16, hkv=4, d=128, cap=64, dtype=torch.bfloat16)
    c["alen"] = torch.tensor([0, 15], dtype=torch.int32)
    c["apath"] = torch.tensor([[0] + [-1] * 15, list(range(16))], dtype=torch.int32)
    lens = _check(c)
    assert (lens - c["ctx"].numpy()).tolist() == [1, 16]


def test_capacity_is_never_exceeded():
    c = _random_case(8, batch=3, n=64, hkv=4, d=128, cap=40, dtype=torch.bfloat16, ctx=[38, 40, 0])
    c["alen"] = torch.tensor([5, 3, 2], dtype=torch.int32)
    c["apath"][:, :6] = torch.arange(6, dtype=torch.int32)
    lens = _check(c)
    assert lens.tolist() == [40, 40, 3]


def test_invalid_entries_and_short_stride():
    c = _random_case(9, batch=3, n=32, hkv=2, d=64, cap=128, dtype=torch.float32, stride=4)
    c["alen"] = torch.tensor([3, 9, -2], dtype=torch.int32)
    c["apath"] = torch.tensor([[0, 5, 99, 7], [0, 1, 2, 3], [0, 1, 2, 3]], dtype=torch.int32)
    before = c["ctx"].numpy().copy()
    lens = _check(c)
    assert (lens - before).tolist() == [2, 4, 0]


def test_two_commits_in_a_row_and_the_accept_outputs():
    """Two rounds on one cache: the second reads the length the first advanced;
    the paths come straight from the GPU acceptance of planted logits."""
    w = W.WORKLOADS["verify_4k"]
    batch, n = 2, 64
    par, tok = W.tree_inputs(w, seed=3, batch=batch)
    logits = W.planted_logits(w, par, tok, seed=3)
    acc = G.glance_greedy_accept(logits.cuda(), par.cuda(), tok.cuda(), path_stride=16)
    c = _random_case(10, batch=batch, n=n, hkv=4, d=128, cap=300, dtype=torch.bfloat16)
    c["alen"], c["apath"] = acc["accept_len"].cpu(), acc["accept_path"].cpu()
    dev = {k: v.cuda() for k, v in c.items()}
    kb, vb = _to_bits(c["k_ctx"]).numpy(), _to_bits(c["v_ctx"]).numpy()
    lens = c["ctx"].numpy()
    for _ in range(2):
        G.glance_commit_path(dev["k_new"], dev["v_new"], dev["alen"], dev["apath"], dev["k_ctx"], dev["v_ctx"],
                             dev["ctx"])
        kb, vb, lens = OC.commit_kv(kb, vb, lens, _to_bits(c["k_new"]).numpy(), _to_bits(c["v_new"]).numpy(),
                                    c["alen"].numpy(), c["apath"].numpy())
    torch.cuda.synchronize()
    np.testing.assert_array_equal(dev["ctx"].cpu().numpy(), lens)
    np.testing.assert_array_equal(_to_bits(dev["k_ctx"].cpu()).numpy(), kb)
    np.testing.assert_array_equal(_to_bits(dev["v_ctx"].cpu()).numpy(), vb)
    assert (lens - c["ctx"].numpy()).tolist() == [2 * (int(a) + 1) for a in c["alen"]]
