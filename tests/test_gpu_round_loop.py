"""Whole GLANCE rounds on the GPU for a tiny fp32 target (Algorithm 1, App. B).

A round runs, on one stream with no host synchronisation inside it: the tree
builder on the drafter's logits, the target's verify pass over the packed tree
(its attention is the library's tree-verify attention over the target's
cache; the dense layers are plain torch), the greedy acceptance with the root
entropy, and the commit of the accepted path into every layer's cache.  The
same round is captured once in a HIP graph and replayed.

Pins: the committed stream equals the target's own greedy autoregressive
decoding (Thm. 1, decided in fp32), graph replays equal eager rounds, the root
entropy matches the float64 entropy of the round's root row, and the caches
end equal to a causal forward's over the committed prefix.  With the sampling
walk in place of the greedy acceptance (temperatures 1 and 0.5), every round's
draws and walk equal the oracle's on the round's own verified logits, and the
caches again equal a causal forward's over what was committed.  The drafter is a
stand-in (no head weights): N(0,1) logits with the true continuation planted
at each offset with probability 0.7, so trees accept some tokens and miss
others.
"""

import numpy as np
import pytest
import torch

import paper_2609_00355_amd as G
from oracle import accept as OA
from oracle import sampling as OS

from gpu_helpers import ensure_lib

pytestmark = pytest.mark.gpu

VOCAB, D_MODEL, LAYERS, HQ, HKV, HD, D_FF = 512, 256, 2, 4, 2, 64, 512
L_DRAFT, BUDGET, PROMPT, N_GEN, CAP = 6, 15, 8, 48, 160


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_lib()


class TinyTarget:
    """Random-weight decoder (RMSNorm, GQA with rotary positions, SwiGLU) in fp32 on the GPU."""

    def __init__(self, seed):
        g = torch.Generator().manual_seed(seed)
        s = 1.0 / np.sqrt(D_MODEL)

        def rnd(*shape, scale):
            return (torch.randn(*shape, generator=g) * scale).cuda()
        self.emb = rnd(VOCAB, D_MODEL, scale=1.0)
        self.layers = []
        for _ in range(LAYERS):
            self.layers.append(dict(
                n1=1.0 + rnd(D_MODEL, scale=0.1), wq=rnd(D_MODEL, HQ * HD, scale=s),
                wk=rnd(D_MODEL, HKV * HD, scale=s), wv=rnd(D_MODEL, HKV * HD, scale=s),
                wo=rnd(HQ * HD, D_MODEL, scale=1.0 / np.sqrt(HQ * HD)), n2=1.0 + rnd(D_MODEL, scale=0.1),
                wg=rnd(D_MODEL, D_FF, scale=s), wu=rnd(D_MODEL, D_FF, scale=s),
                wd=rnd(D_FF, D_MODEL, scale=1.0 / np.sqrt(D_FF))))
        self.nf = 1.0 + rnd(D_MODEL, scale=0.1)
        self.head = rnd(D_MODEL, VOCAB, scale=4.0 * s)
        half = HD // 2
        self.inv = (10000.0 ** (-torch.arange(half, dtype=torch.float32) * 2.0 / HD)).cuda()

    @staticmethod
    def norm(x, gain):
        return x * torch.rsqrt((x * x).mean(-1, keepdim=True) + 1e-6) * gain

    def rope(self, x, pos):  # x [T][H][D], pos [T] (device)
        ang = pos.float()[:, None] * self.inv[None, :]
        c, s = torch.cos(ang)[:, None, :], torch.sin(ang)[:, None, :]
        h = HD // 2
        return torch.cat([x[..., :h] * c - x[..., h:] * s, x[..., :h] * s + x[..., h:] * c], dim=-1)

    def qkv(self, lw, h, pos):
        x = self.norm(h, lw["n1"])
        t = h.shape[0]
        q = self.rope((x @ lw["wq"]).view(t, HQ, HD), pos)
        k = self.rope((x @ lw["wk"]).view(t, HKV, HD), pos)
        return q, k, (x @ lw["wv"]).view(t, HKV, HD)

    def mlp(self, lw, h, o):
        h = h + o.reshape(h.shape[0], -1) @ lw["wo"]
        x = self.norm(h, lw["n2"])
        gate = x @ lw["wg"]
        return h + (gate * torch.sigmoid(gate) * (x @ lw["wu"])) @ lw["wd"]

    def logits(self, h):
        return self.norm(h, self.nf) @ self.head

    def forward_causal(self, tokens):
        """Plain torch causal pass: logits [T][V] and per-layer K, V [T][Hkv][D]."""
        t = len(tokens)
        pos = torch.arange(t, device="cuda")
        h = self.emb[torch.as_tensor(tokens, device="cuda")]
        mask = torch.ones(t, t, dtype=torch.bool, device="cuda").tril()
        kv = []
        for lw in self.layers:
            q, k, v = self.qkv(lw, h, pos)
            kv.append((k, v))
            kk = k.repeat_interleave(HQ // HKV, dim=1)
            vv = v.repeat_interleave(HQ // HKV, dim=1)
            s = torch.einsum("ihd,jhd->hij", q, kk) / np.sqrt(HD)
            s = s.masked_fill(~mask[None], float("-inf"))
            o = torch.einsum("hij,jhd->ihd", torch.softmax(s, dim=-1), vv)
            h = self.mlp(lw, h, o)
        return self.logits(h), kv


def greedy_ar(m, prompt, n):
    seq, margins = list(prompt), []
    for _ in range(n):
        lg, _ = m.forward_causal(seq)
        row = lg[-1].double().cpu().numpy()
        top = np.sort(row)[-2:]
        margins.append(top[1] - top[0])
        seq.append(int(np.argmax(row)))
    return seq[len(prompt):], min(margins)


class Decoder:
    """Buffers, prepared library calls and the round of one sequence."""

    def __init__(self, m, prompt, temperature=None, seed=0, device_round=False):
        self.m = m
        self.temperature, self.seed, self.round_no = temperature, seed, 0
        # with device_round the sampling call reads and advances a device
        # counter, so a captured round draws fresh noise on every replay
        self.round_counter = torch.zeros(1, dtype=torch.int32, device="cuda") if device_round else None
        n = BUDGET + 1
        self.kc = torch.zeros(LAYERS, HKV, CAP, HD, device="cuda")
        self.vc = torch.zeros_like(self.kc)
        lg, kv = m.forward_causal(prompt)                       # prefill
        for li, (k, v) in enumerate(kv):
            self.kc[li, :, :len(prompt)] = k.transpose(0, 1)
            self.vc[li, :, :len(prompt)] = v.transpose(0, 1)
        self.ctx = torch.full((LAYERS,), len(prompt), dtype=torch.int32, device="cuda")
        self.root = lg[-1].argmax().view(1).to(torch.int32)
        self.draft = torch.zeros(1, L_DRAFT, VOCAB, device="cuda")
        self.out = torch.full((N_GEN + 64,), -1, dtype=torch.int32, device="cuda")
        self.out[0] = self.root[0]
        self.count = torch.ones(1, dtype=torch.int64, device="cuda")
        self.entropy_log = []
        # fixed outputs and workspaces; the calls take the current stream each time
        # (the capture stream while a graph is recorded)
        self.tree_out = {"parents": torch.zeros(1, n, dtype=torch.int32, device="cuda"),
                         "tokens": torch.zeros(1, n, dtype=torch.int32, device="cuda"), "scores": None}
        self.tree_ws = torch.empty(G.glance_tree_workspace_size(1, L_DRAFT, VOCAB, BUDGET), dtype=torch.uint8,
                                   device="cuda")
        self.parents, self.tokens = self.tree_out["parents"], self.tree_out["tokens"]
        self.logits_buf = torch.zeros(1, n, VOCAB, device="cuda")
        self.acc = G.glance_greedy_accept(self.logits_buf, self.parents, self.tokens, path_stride=16,
                                          want_entropy=True)
        self.acc_ws = torch.zeros(G.glance_accept_workspace_size(1, n, VOCAB), dtype=torch.uint8, device="cuda")
        if temperature is not None:  # the sampling walk writes draws in place of argmax rows
            self.acc = {"draws": torch.zeros(1, n, dtype=torch.int32, device="cuda"),
                        "accept_len": torch.zeros(1, dtype=torch.int32, device="cuda"),
                        "accept_path": torch.zeros(1, 16, dtype=torch.int32, device="cuda"),
                        "next_root": torch.zeros(1, dtype=torch.int32, device="cuda")}
        self.k_new = torch.zeros(LAYERS, n, HKV, HD, device="cuda")
        self.v_new = torch.zeros_like(self.k_new)
        self.alen_l = torch.zeros(LAYERS, dtype=torch.int32, device="cuda")
        self.apath_l = torch.zeros(LAYERS, 16, dtype=torch.int32, device="cuda")
        self.ar_idx = torch.arange(16, device="cuda")

    def round(self):
        m = self.m
        G.glance_build_tree(self.draft, self.root, BUDGET, outputs=self.tree_out,
                            workspace=self.tree_ws)             # tree from the drafter's logits
        par, tok = self.parents[0].long(), self.tokens[0].long()
        depth = torch.zeros_like(par)
        for _ in range(L_DRAFT):                                # depth by repeated parent lookups
            depth = torch.where(par >= 0, depth[par.clamp(min=0)] + 1, torch.zeros_like(depth))
        pos = self.ctx[0].long() + depth
        h = m.emb[tok]
        for li, lw in enumerate(m.layers):                      # verify pass over the packed tree
            q, k, v = m.qkv(lw, h, pos)
            self.k_new[li].copy_(k)
            self.v_new[li].copy_(v)
            o, _ = G.glance_tree_verify_attn(q[None].contiguous(), self.kc[li:li + 1], self.vc[li:li + 1],
                                             self.k_new[li:li + 1], self.v_new[li:li + 1], self.ctx[0:1],
                                             self.parents, want_lse=False)
            h = m.mlp(lw, h, o[0])
        self.logits_buf.copy_(m.logits(h)[None])
        if self.temperature is None:
            G.glance_greedy_accept(self.logits_buf, self.parents, self.tokens, path_stride=16, outputs=self.acc,
                                   workspace=self.acc_ws, want_entropy=True)  # argmax, walk, root entropy
        else:                                                   # draws at temperature T, walk
            G.glance_sample_accept(self.logits_buf, self.parents, self.tokens, self.temperature, self.seed,
                                   0 if self.round_counter is not None else self.round_no, path_stride=16,
                                   outputs=self.acc, workspace=self.acc_ws, round_counter=self.round_counter)
        self.alen_l.copy_(self.acc["accept_len"].expand(LAYERS))
        self.apath_l.copy_(self.acc["accept_path"].expand(LAYERS, 16))
        G.glance_commit_path(self.k_new, self.v_new, self.alen_l, self.apath_l, self.kc, self.vc, self.ctx)
        a = self.acc["accept_len"][0].long()
        path = self.acc["accept_path"][0].long()
        toks = torch.where(self.ar_idx < a, self.tokens[0][path.clamp(min=0)].roll(-1), -1)
        toks = torch.where(self.ar_idx == a, self.acc["next_root"][0], toks)
        idx = (self.count + self.ar_idx).clamp(max=self.out.numel() - 1)
        keep = self.ar_idx <= a
        self.out.index_put_((idx,), torch.where(keep, toks.int(), self.out[idx]))
        self.count += a + 1
        self.root.copy_(self.acc["next_root"])

    def set_draft_tokens(self, cont, seed):
        """The stand-in drafter planting the given continuation of the root at every offset."""
        rng = np.random.default_rng(seed)
        z = rng.normal(size=(L_DRAFT, VOCAB)).astype(np.float32)
        for j, t in enumerate(cont[:L_DRAFT]):
            z[j, t] = 8.0
        self.draft.copy_(torch.from_numpy(z)[None])

    def set_draft(self, ar_stream, prompt, seed):
        """The stand-in drafter: N(0,1) logits, the true continuation planted with p = 0.7."""
        c = int(self.count.item())                              # tokens generated so far (root included)
        rng = np.random.default_rng(seed)
        z = rng.normal(size=(L_DRAFT, VOCAB)).astype(np.float32)
        for j in range(L_DRAFT):
            if c + j < len(ar_stream) and rng.uniform() < 0.7:
                z[j, ar_stream[c + j]] = 8.0
        self.draft.copy_(torch.from_numpy(z)[None])


def _setup():
    for seed in range(10):
        m = TinyTarget(seed)
        prompt = np.random.default_rng(seed + 7).integers(0, VOCAB, size=PROMPT).tolist()
        ar, margin = greedy_ar(m, prompt, N_GEN + 1)
        if margin > 2e-3:
            return m, prompt, ar
    pytest.fail("no seed with a clear argmax margin")


@pytest.fixture(scope="module")
def setup():
    return _setup()


def _decode(m, prompt, ar, graph):
    d = Decoder(m, prompt)
    rounds, entropies = 0, []
    g = None
    while int(d.count.item()) < N_GEN:
        d.set_draft(ar, prompt, seed=rounds)
        if graph and g is None and rounds == 1:                 # capture after one eager round
            torch.cuda.synchronize()
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.current_stream())
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=s):
                d.round()
            torch.cuda.synchronize()
            # capture recorded the work without running it: run this round for real
            g.replay()
        elif g is not None:
            g.replay()
        else:
            d.round()
        torch.cuda.synchronize()
        row0 = d.logits_buf[0, 0].double().cpu().numpy()
        entropies.append((float(d.acc["root_entropy"][0]), OA.row_entropy(row0)))
        rounds += 1
        assert rounds < 200
    out = d.out[:N_GEN].cpu().tolist()
    return out, d, entropies, rounds


def test_rounds_commit_the_greedy_stream(setup):
    m, prompt, ar = setup
    out, d, ents, rounds = _decode(m, prompt, ar, graph=False)
    assert out == ar[:N_GEN]
    assert rounds < N_GEN - 5                                    # trees were accepted, not just roots
    for h, ref in ents:
        assert abs(h - ref) <= 2e-4 + 2e-5 * abs(ref)
    # the caches hold exactly the causal pass's keys and values of the committed prefix
    ctx = int(d.ctx[0])
    assert (d.ctx == ctx).all() and ctx == PROMPT + int(d.count.item()) - 1
    _, kv = m.forward_causal(prompt + out[:ctx - PROMPT])
    for li, (k, v) in enumerate(kv):
        torch.testing.assert_close(d.kc[li, :, :ctx], k.transpose(0, 1), rtol=1e-4, atol=1e-4)
        torch.testing.assert_close(d.vc[li, :, :ctx], v.transpose(0, 1), rtol=1e-4, atol=1e-4)


def test_graph_replays_equal_eager_rounds(setup):
    m, prompt, ar = setup
    eager, _, _, r1 = _decode(m, prompt, ar, graph=False)
    graphed, _, ents, r2 = _decode(m, prompt, ar, graph=True)
    assert graphed == eager == ar[:N_GEN]
    assert r1 == r2
    for h, ref in ents:
        assert abs(h - ref) <= 2e-4 + 2e-5 * abs(ref)


@pytest.mark.parametrize("temperature,graph", [(1.0, False), (0.5, False), (1.0, True)])
def test_sampling_rounds_follow_the_oracle_walk(setup, temperature, graph):
    """Whole rounds with the sampling walk, eagerly with the round number as a
    call argument, or captured once in a HIP graph and replayed with a device
    round counter (so each replay draws the next round's noise): every
    round's draws, accepted length and path and next root equal the oracle's
    sampling walk on the GPU's own verified logits, the committed tokens are
    the walk's, and the caches end equal to a causal pass over the committed
    prefix."""
    m, prompt, ar = setup
    seed = 4242
    d = Decoder(m, prompt, temperature=temperature, seed=seed, device_round=graph)
    committed = [int(d.root[0])]
    accepted = 0
    g = None
    while int(d.count.item()) < N_GEN:
        # the drafter proposes the greedy continuation of what was committed so
        # far (the root included), which draws at these temperatures often follow
        cont, _ = greedy_ar(m, prompt + committed, L_DRAFT)
        d.set_draft_tokens(cont, seed=d.round_no)
        if graph and g is None and d.round_no == 1:            # capture after one eager round
            torch.cuda.synchronize()
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=side):
                d.round()
            torch.cuda.synchronize()
            g.replay()
        elif g is not None:
            g.replay()
        else:
            d.round()
        torch.cuda.synchronize()
        if graph:
            assert int(d.round_counter.item()) == d.round_no + 1
        rows = d.logits_buf[0].cpu().numpy()
        par, tok = d.parents[0].cpu().tolist(), d.tokens[0].cpu().tolist()
        draws, a, path, nr = OS.sampling_walk(rows, par, tok, temperature, seed, d.round_no, 0)
        assert d.acc["draws"][0].cpu().tolist() == draws, d.round_no
        assert int(d.acc["accept_len"][0]) == a
        assert d.acc["accept_path"][0].cpu().tolist()[:a + 1] == list(path)
        assert int(d.acc["next_root"][0]) == nr
        committed += [tok[c] for c in path[1:]] + [nr]
        accepted += a
        d.round_no += 1
        assert d.round_no < 200
    out = d.out[:N_GEN].cpu().tolist()
    assert out == committed[:N_GEN]
    assert accepted >= 10                                        # drafted tokens were drawn and kept
    ctx = int(d.ctx[0])
    assert ctx == PROMPT + int(d.count.item()) - 1
    _, kv = m.forward_causal(prompt + committed[:ctx - PROMPT])
    for li, (k, v) in enumerate(kv):
        torch.testing.assert_close(d.kc[li, :, :ctx], k.transpose(0, 1), rtol=1e-4, atol=1e-4)
        torch.testing.assert_close(d.vc[li, :, :ctx], v.transpose(0, 1), rtol=1e-4, atol=1e-4)
    print(f"[T={temperature} graph={graph}] rounds={d.round_no} accepted={accepted}", flush=True)
