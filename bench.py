"""Benchmark of one GLANCE decode round on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input:
block-draft attention, then tree-verify attention, then greedy acceptance
(vocabulary argmax of every verified row and the walk), back to back on one
stream, replayed from a HIP graph captured once per input set (--eager: the
prepared C-ABI calls one by one).  The headline workload is the grounded
long-document configuration: batch 4, 28 query / 4 KV heads, head_dim 128,
bf16, 16384 context tokens per sequence (14336 image + 2048 text), a 16-row
draft block and a 64-row tree, verified rows over a 152064-token vocabulary.

Inputs are resident in HBM before timing starts.  Several copies of the input
set rotate from step to step so that each step's context reads miss the
256 MB last-level cache ("cold"; a doc_16k step reads about 350 MB); the
"warm" figure replays one set, so whatever fits stays cached.  The draft and
the verify read separate caches (the draft head's and the target's).

Prints one JSON line per configuration: first the smaller configurations
(tiny fp32, the 2k draft, the 4k verify, the ragged serving mix), each with
its own round latency, p10/p90 over the timed steps, warm and cold, and the
float64 oracle timed on a bounded sample; the last line is the headline
(doc_16k): whole-round latency (value, from the wall clock over the timed
steps), per-kernel times from HIP events recorded on the library's stream,
the roofline of the dominant kernel and the oracle's time.
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak
# Vector ALU issue peak: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz = 39.3e12
# full-rate lane operations per second (a 32x32 -> 64-bit multiply issues at
# a quarter of that rate and counts as 4).
VALU_PEAK_TOPS = 39.32
# Work of the sampling walk's row draws per token, in full-rate lane
# operations: a quarter of one Philox4x32-10 call (20 64-bit multiplies at 4
# each plus 20 three-input XORs: 100 per four tokens = 25), the noise bound and
# its test (8), and the load and unpack of a bf16 pair (1).
SAMPLE_OPS_PER_TOKEN = 34


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="doc_16k", help="the headline workload (last line)")
    ap.add_argument("--configs", default="tiny_fp32,draft_2k,verify_4k,ragged_mix",
                    help="workloads timed before the headline, one line each ('' for none)")
    ap.add_argument("--eager", action="store_true", help="launch the prepared calls one by one (no HIP graph)")
    ap.add_argument("--sets", type=int, default=4, help="input copies rotated across steps")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="budget of the headline's oracle timing")
    ap.add_argument("--cpu-seconds-config", type=float, default=4.0,
                    help="budget of each smaller configuration's oracle timing")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 256 MiB device copy (reference for HBM byte counters)")
    ap.add_argument("--no-tree", action="store_true", help="skip the tree-builder measurement")
    ap.add_argument("--verify-sweep", action="store_true",
                    help="instead of the round, time the tree-verify attention alone at tree widths "
                         "16, 32, 48 and 64 (one JSON line each) and exit")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarise two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of this bench "
                         "with --calibrate-copy into profiles/traffic.json, then exit")
    return ap.parse_args()


def kv_bytes(w, ctx_lens):
    return int(sum(int(c) for c in ctx_lens)) * w.hkv * w.d * 2 * 2  # K and V, bf16


def attn_flops(w, ctx_lens, n, visible_new):
    """4*D flops (Q.K and P.V) per (query head, row, visible key)."""
    ctx_rows = sum(int(c) for c in ctx_lens) * n
    return 4.0 * w.d * w.hq * (ctx_rows + visible_new)


def tree_visible_pairs(parents):
    """sum over nodes of |ancestors-or-self| (the visible tree keys of the verify)."""
    tot = 0
    for par in parents:
        par = [int(x) for x in par]
        for i in range(len(par)):
            j = i
            while j >= 0:
                tot += 1
                j = par[j]
    return tot


def source_hash(path):
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def load_traffic(kernel_key, src, workload):
    """HBM bytes per launch measured with rocprofv3 counters, if taken on the current source and
    on this workload (the counter runs time one workload)."""
    p = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(p):
        return None
    try:
        allrec = json.load(open(p))
    except Exception:
        return None
    rec = allrec.get(kernel_key)
    if not rec or rec.get("source_sha") != source_hash(src) or allrec.get("workload", "doc_16k") != workload:
        return None
    return rec.get("bytes_per_launch")


COPY_BYTES = 256 << 20
COPY_KERNEL = "neg_kernel"  # the calibration copy: out = -in over COPY_BYTES of fp32
KERNEL_KEYS = {"draft": "attn_bf16<128, false", "verify": "attn_bf16<128, true",
               "accept": "argmax_partial<true, true>", "tree_scan": "tree_scan<true>",
               "tree_rank": "tree_rank<true>", "tree_enum": "tree_enum",
               "sample": "sample_partial<true, true>"}
KERNEL_SRC = {"draft": "attn_bf16.hip", "verify": "attn_bf16.hip", "accept": "accept.hip",
              "tree_scan": "tree.hip", "tree_rank": "tree.hip", "tree_enum": "tree.hip",
              "sample": "accept.hip"}


def summarise_traffic(fetch_dir, write_dir, workload):
    """Per-launch HBM bytes of the round's main kernels from rocprofv3 counter CSVs.

    FETCH_SIZE and WRITE_SIZE read KiB per dispatch; each is scaled by the
    ratio between the bytes a plain streaming kernel over COPY_BYTES really
    moves (reads COPY_BYTES, writes COPY_BYTES) and what the same counter
    reports for it.
    """
    import csv
    import glob

    def load(d, counter):
        per = {}
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            for r in csv.DictReader(open(f)):
                if r["Counter_Name"] != counter:
                    continue
                per.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return per

    fetch, write = load(fetch_dir, "FETCH_SIZE"), load(write_dir, "WRITE_SIZE")

    def avg(per, key):
        vals = [v for k, vs in per.items() if key in k for v in vs]
        return sum(vals) / len(vals) if vals else None

    f_copy, w_copy = avg(fetch, COPY_KERNEL), avg(write, COPY_KERNEL)
    if not f_copy or not w_copy:
        raise SystemExit("no copy-kernel reading in the counter runs (use --calibrate-copy)")
    f_scale, w_scale = COPY_BYTES / (f_copy * 1024), COPY_BYTES / (w_copy * 1024)
    out = {"workload": workload, "copy_bytes": COPY_BYTES, "fetch_scale": round(f_scale, 4),
           "write_scale": round(w_scale, 4)}
    for name, key in KERNEL_KEYS.items():
        f, w = avg(fetch, key), avg(write, key)
        if f is None or w is None:
            continue
        src = os.path.join(ROOT, "paper_2609_00355_amd", "csrc", KERNEL_SRC[name])
        out[name] = {"kernel": key, "source_sha": source_hash(src),
                     "fetch_bytes": round(f * 1024 * f_scale), "write_bytes": round(w * 1024 * w_scale),
                     "bytes_per_launch": round((f * 1024 * f_scale) + (w * 1024 * w_scale))}
    path = os.path.join(ROOT, "profiles", "traffic.json")
    json.dump(out, open(path, "w"), indent=1)
    print(json.dumps(out))


def host_info():
    """Host cores and CPU model for the oracle timing."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        nproc = len(os.sched_getaffinity(0))
    except AttributeError:
        nproc = os.cpu_count() or 1
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        threads = nproc
    return {"nproc": int(nproc), "cpu_model": model, "blas_threads": int(threads)}


def cpu_baseline(inputs, budget_s):
    """The float64 oracle, as it stands, on a bounded sample of the same round:
    whole sequences (every step of the workload for one sequence), round after
    round, until the time budget is spent; the rate is scaled to one round by
    context tokens."""
    from oracle import accept as OA
    from oracle import attention as OT
    w = inputs["workload"]
    info = host_info()
    ctx = [int(c) for c in inputs["ctx_lens"]]
    t0 = time.perf_counter()
    done, tok_done = 0, 0
    while True:
        b = done % w.batch
        sl = slice(b, b + 1)
        if "draft" in w.steps:
            d = inputs["draft"]
            OT.block_draft_attn(d["q"][sl], d["k_ctx"][sl], d["v_ctx"][sl], d["k_new"][sl], d["v_new"][sl],
                                d["ctx_lens"][sl])
        if "verify" in w.steps:
            v = inputs["verify"]
            OT.tree_verify_attn(v["q"][sl], v["k_ctx"][sl], v["v_ctx"][sl], v["k_new"][sl], v["v_new"][sl],
                                v["ctx_lens"][sl], inputs["parents"][sl])
        if "accept" in w.steps:
            OA.greedy_accept(inputs["logits"][sl], inputs["parents"][sl], inputs["tokens"][sl])
        done += 1
        tok_done += ctx[b] + 1
        if time.perf_counter() - t0 > budget_s:
            break
    dt = time.perf_counter() - t0
    per_round_us = dt * (sum(ctx) + w.batch) / tok_done * 1e6
    return {"value": round(per_round_us, 1), "unit": "us per round", "cores": info["blas_threads"],
            "nproc": info["nproc"], "cpu_model": info["cpu_model"], "kind": "oracle",
            "sample": f"{done} sequence passes ({done / w.batch:.2f} rounds) of {w.name} ({' + '.join(w.steps)}, "
                      f"numpy float64), scaled to one round by context tokens; {dt:.1f} s"}


def verify_sweep(args, w, G, C, torch, np, dev):
    """Verify attention cost against tree width at the workload's context: the
    same context for every width, a best-first tree of n rows per sequence."""
    ctx = C.context_lengths(w)
    for n in (16, 32, 48, 64):
        sets = []
        for r in range(args.sets):
            inp = C.attention_inputs(w, "verify", n, ctx, seed=r)
            par, _ = C.tree_inputs(w, r, "best_first", n=n, batch=w.batch)
            vv = {k: (t.to(dev) if torch.is_tensor(t) else t) for k, t in inp.items()}
            call, out, _ = G.prepare_tree_verify_attn(vv["q"], vv["k_ctx"], vv["v_ctx"], vv["k_new"],
                                                      vv["v_new"], vv["ctx_lens"], par.to(dev))
            sets.append((call, vv, par, out))
        torch.cuda.synchronize()
        for i in range(args.warmup):
            sets[i % len(sets)][0]()
        reps = max(args.steps, 20)
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, b in evs:
            a.record()
            b.record()
        torch.cuda.synchronize()
        for i in range(reps):
            G.glance_set_kernel_events(*evs[i])
            sets[i % len(sets)][0]()
        torch.cuda.synchronize()
        us = float(np.median([a.elapsed_time(b) for a, b in evs]) * 1e3)
        par0 = sets[0][2]
        vis = tree_visible_pairs(par0.numpy())
        fl = attn_flops(w, ctx, n, vis)
        kvb = kv_bytes(w, ctx)
        print(json.dumps({"mode": "verify_sweep", "workload": w.name, "tree_rows": n, "us": round(us, 2),
                          "tflops": round(fl / us / 1e6, 1), "mfma_frac": round(fl / us / 1e6 / MFMA_BF16_PEAK_TFLOPS, 3),
                          "kv_gbps": round(kvb / us / 1e3, 1)}), flush=True)
        del sets
        torch.cuda.empty_cache()


def measure_tree_builder(args, w, G, C, torch, np, dev, stream):
    """The tree builder (Algorithm 1, second step) on the drafter's logits of the
    same workload: 15 offsets x vocab per sequence, budget 63.  Timed on its own
    (it is not one of the round's attention / acceptance kernels): HIP events
    around its three kernels, median over the steps, rotating input copies."""
    budget = w.n_tree - 1
    calls = []
    for r in range(args.sets):
        zd = C.draft_logits(w, 0).to(dev)
        roots = C.draft_roots(w, 0).to(dev)
        call, out = G.prepare_build_tree(zd, roots, budget, want_scores=False)
        calls.append((call, out, zd, roots))
    for i in range(args.warmup):
        calls[i % len(calls)][0]()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    for a, b in evs:
        a.record(stream)
        b.record(stream)
    torch.cuda.synchronize()
    for i in range(args.steps):
        G.glance_set_kernel_events(*evs[i])
        calls[i % len(calls)][0]()
    torch.cuda.synchronize()
    us = float(np.median([a.elapsed_time(b) for a, b in evs]) * 1e3)
    nbytes = w.batch * (w.n_draft - 1) * w.vocab * 2
    gbps = nbytes / us / 1e3
    depth = []
    par = calls[0][1]["parents"].cpu().numpy()
    for b in range(par.shape[0]):
        d = [0] * par.shape[1]
        for i in range(1, par.shape[1]):
            d[i] = d[par[b, i]] + 1
        depth.append(max(d))
    src = os.path.join(ROOT, "paper_2609_00355_amd", "csrc", "tree.hip")
    parts = [load_traffic(k, src, w.name) for k in ("tree_scan", "tree_rank", "tree_enum")]
    traffic = sum(parts) if all(t is not None for t in parts) else None
    return {"us": round(us, 2), "kernels": "tree_scan + tree_rank + tree_enum",
            "input": f"drafter logits {w.batch} x {w.n_draft - 1} x {w.vocab} bf16, budget {budget}",
            "gbps": round(gbps, 1), "bound": "hbm", "frac": round(gbps / HBM_PEAK_GBS, 4),
            "traffic": traffic, "tree_depth": depth}


def measure_commit(args, w, s, G, torch, np, dev, stream, ctx):
    """The commit of the round's accepted paths (root + accepted nodes' keys and
    values of the verify pass appended to a cache with room for them), timed
    with HIP events around its kernel; the lengths are reset between calls
    outside the timed interval."""
    vv = s["keep"]["verify"][0]
    k_new, v_new = vv["k_new"], vv["v_new"]
    a_out = s["a_out"]
    cap = int(max(ctx)) + w.n_tree
    k_ctx = torch.zeros((w.batch, w.hkv, cap, w.d), dtype=k_new.dtype, device=dev)
    v_ctx = torch.zeros_like(k_ctx)
    lens0 = torch.as_tensor(np.asarray(ctx, dtype=np.int32)).to(dev)
    lens = lens0.clone()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    for a, b in evs:
        a.record(stream)
        b.record(stream)
    for i in range(args.warmup + args.steps):
        lens.copy_(lens0)
        if i >= args.warmup:
            G.glance_set_kernel_events(*evs[i - args.warmup])
        G.glance_commit_path(k_new, v_new, a_out["accept_len"], a_out["accept_path"], k_ctx, v_ctx, lens,
                             stream=stream)
    torch.cuda.synchronize()
    us = float(np.median([a.elapsed_time(b) for a, b in evs]) * 1e3)
    rows = int((a_out["accept_len"].cpu().numpy() + 1).sum())
    nbytes = rows * w.hkv * w.d * k_new.element_size() * 2 * 2  # K and V, read and written
    return {"us": round(us, 2), "kernel": "commit_kernel", "rows": rows, "bytes": nbytes,
            "bound": "launch latency (a few KB per call)"}


def measure_sample(args, w, sets, G, torch, np, stream):
    """The sampling walk at temperature 1 (glance_sample_accept) on the round's
    verified logits, in place of the greedy acceptance: HIP events around its
    row-draw kernel, mean over the steps, the round number advancing every call
    so every call draws fresh noise."""
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    for a, b in evs:
        a.record(stream)
        b.record(stream)
    outs = []
    for s in sets:
        logits, par, tok = s["keep"]["logits"], s["keep"]["par"], s["keep"]["tok"]
        outs.append(G.glance_sample_accept(logits, par, tok, 1.0, 2026, 0, path_stride=16, stream=stream))
    torch.cuda.synchronize()
    for i in range(args.warmup + args.steps):
        s = sets[i % len(sets)]
        logits, par, tok = s["keep"]["logits"], s["keep"]["par"], s["keep"]["tok"]
        if i >= args.warmup:
            G.glance_set_kernel_events(*evs[i - args.warmup])
        G.glance_sample_accept(logits, par, tok, 1.0, 2026, i + 1, path_stride=16,
                               outputs=outs[i % len(sets)], stream=stream)
    torch.cuda.synchronize()
    us = float(np.mean([a.elapsed_time(b) for a, b in evs]) * 1e3)
    tokens = w.batch * w.n_tree * w.vocab
    nbytes = tokens * 2
    acc = outs[0]["accept_len"].cpu().numpy()
    ops = tokens * SAMPLE_OPS_PER_TOKEN
    return {"us": round(us, 2), "kernel": "sample_partial<true,true>",
            "input": f"verified logits {w.batch} x {w.n_tree} x {w.vocab} bf16, T = 1",
            "gtokens_per_s": round(tokens / us / 1e3, 1), "gbps": round(nbytes / us / 1e3, 1),
            "hbm_frac": round(nbytes / us / 1e3 / HBM_PEAK_GBS, 4), "bound": "alu",
            "alu_ops_per_token": SAMPLE_OPS_PER_TOKEN, "achieved_tops": round(ops / us / 1e6, 2),
            "peak_tops": VALU_PEAK_TOPS, "frac": round(ops / us / 1e6 / VALU_PEAK_TOPS, 4),
            "traffic": load_traffic("sample", os.path.join(ROOT, "paper_2609_00355_amd", "csrc", "accept.hip"),
                                    w.name),
            "mean_accept_len": round(float(acc.mean()), 3)}


HEADLINE_METRIC = "draft+verify round latency (\u00b5s) and achieved KV HBM GB/s at 16k ctx, 1 MI355X"


def prepare_sets(w, n_sets, G, C, torch, dev):
    """Device copies of one round's inputs and the prepared calls of the
    workload's steps, n_sets times (all copies hold the same values)."""
    inputs = C.round_inputs(w, seed=0)
    sets = []
    for _ in range(n_sets):
        s = {"calls": {}, "keep": {}}
        if "verify" in w.steps or "accept" in w.steps:
            s["keep"]["par"] = inputs["parents"].to(dev)
            s["keep"]["tok"] = inputs["tokens"].to(dev)
        if "draft" in w.steps:
            dd = {k: t.to(dev) for k, t in inputs["draft"].items()}
            call, out, _ = G.prepare_block_draft_attn(dd["q"], dd["k_ctx"], dd["v_ctx"], dd["k_new"], dd["v_new"],
                                                      dd["ctx_lens"])
            s["calls"]["draft"], s["keep"]["draft"] = call, (dd, out)
        if "verify" in w.steps:
            vv = {k: t.to(dev) for k, t in inputs["verify"].items()}
            call, out, _ = G.prepare_tree_verify_attn(vv["q"], vv["k_ctx"], vv["v_ctx"], vv["k_new"], vv["v_new"],
                                                      vv["ctx_lens"], s["keep"]["par"])
            s["calls"]["verify"], s["keep"]["verify"] = call, (vv, out)
        if "accept" in w.steps:
            logits = inputs["logits"].to(dev)
            call, a_out = G.prepare_greedy_accept(logits, s["keep"]["par"], s["keep"]["tok"], path_stride=16)
            s["calls"]["accept"], s["keep"]["logits"], s["a_out"] = call, logits, a_out
        sets.append(s)
    return inputs, sets


def run_step(s):
    for name in ("draft", "verify", "accept"):
        if name in s["calls"]:
            s["calls"][name]()


def time_rounds(args, sets, stream, torch, np):
    """Round latency: the wall clock over exactly args.steps steps (rotating
    the input sets), then per-step HIP events for p10/p50/p90 (cold: rotating
    sets; warm: one set)."""
    graphs = None
    if not args.eager:
        graphs = []
        for s in sets:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=stream):
                run_step(s)
            graphs.append(g)
        torch.cuda.synchronize()

    def run(i, rotate=True):
        k = i % len(sets) if rotate else 0
        if graphs:
            graphs[k].replay()
        else:
            run_step(sets[k])

    for i in range(args.warmup):
        run(i)
    torch.cuda.synchronize()
    # ---- timed region: exactly K steps, synchronised on both sides
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        run(i)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    def per_step(rotate):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
        for i, (a, b) in enumerate(evs):
            a.record(stream)
            run(i, rotate)
            b.record(stream)
        torch.cuda.synchronize()
        us = np.array([a.elapsed_time(b) * 1e3 for a, b in evs])
        return [round(float(np.percentile(us, q)), 2) for q in (10, 50, 90)]

    cold = per_step(True)
    warm = per_step(False)
    return {"wall_us": wall / args.steps * 1e6, "wall_s": wall, "cold": cold, "warm": warm,
            "launch": "HIP graph replay (one graph per input set)" if graphs else "eager (prepared C-ABI calls)"}


def kernel_times(args, sets, stream, G, torch, np):
    """Per step of the round: the main kernel alone (HIP events the library
    records around it on its stream) and the whole call (events around the
    call: attention + merge pass, argmax + walk), eager, rotating sets."""
    names = [k for k in ("draft", "verify", "accept") if k in sets[0]["calls"]]
    reps = max(args.steps, 10)
    ev = lambda: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    kern = {k: [ev() for _ in range(reps)] for k in names}
    call = {k: [ev() for _ in range(reps)] for k in names}
    for pairs in list(kern.values()) + list(call.values()):
        for a, b in pairs:  # torch creates the HIP events lazily, at first record
            a.record(stream)
            b.record(stream)
    torch.cuda.synchronize()
    for i in range(reps):
        s = sets[i % len(sets)]
        for k in names:
            G.glance_set_kernel_events(*kern[k][i])
            call[k][i][0].record(stream)
            s["calls"][k]()
            call[k][i][1].record(stream)
    torch.cuda.synchronize()
    med = lambda pairs: float(np.median([a.elapsed_time(b) * 1e3 for a, b in pairs]))
    return {k: med(kern[k]) for k in names}, {k: med(call[k]) for k in names}


def round_work(w, inputs):
    """Algorithmic bytes and flops of each step of one round."""
    ctx = inputs["ctx_lens"]
    kvb = kv_bytes(w, ctx) if w.dtype == "bf16" else kv_bytes(w, ctx) * 2
    esz = 2 if w.dtype == "bf16" else 4
    work = {}
    if "draft" in w.steps:
        qo = w.batch * w.n_draft * (w.hq + w.hkv) * w.d * esz * 2
        work["draft"] = {"bytes": kvb + qo, "flops": attn_flops(w, ctx, w.n_draft, w.batch * w.n_draft * w.n_draft)}
    if "verify" in w.steps:
        qo = w.batch * w.n_tree * (w.hq + w.hkv) * w.d * esz * 2
        vis = tree_visible_pairs(inputs["parents"].numpy())
        work["verify"] = {"bytes": kvb + qo, "flops": attn_flops(w, ctx, w.n_tree, vis)}
    if "accept" in w.steps:
        work["accept"] = {"bytes": w.batch * w.n_tree * w.vocab * esz, "flops": 0.0}
    return work, kvb


def per_kernel_report(w, work, k_us, c_us):
    mfma_peak = MFMA_BF16_PEAK_TFLOPS if w.dtype == "bf16" else None
    out = {}
    for k in k_us:
        gbps = work[k]["bytes"] / k_us[k] / 1e3
        rec = {"us": round(k_us[k], 2), "call_us": round(c_us[k], 2), "gbps": round(gbps, 1)}
        if k == "accept":
            rec.update(kernel="argmax_partial", bound="hbm", frac=round(gbps / HBM_PEAK_GBS, 3))
        else:
            tf = work[k]["flops"] / k_us[k] / 1e6
            rec["tflops"] = round(tf, 1)
            rec["kernel"] = f"attn_bf16<{w.d},{'true' if k == 'verify' else 'false'}>" if w.dtype == "bf16" \
                else f"attn_f32<{w.d},{'true' if k == 'verify' else 'false'}>"
            if k == "verify" and mfma_peak:
                rec.update(bound="mfma", frac=round(tf / mfma_peak, 3))
            else:
                rec.update(bound="hbm", frac=round(gbps / HBM_PEAK_GBS, 3))
        out[k] = rec
    return out


def describe(w, inputs):
    import numpy as np
    ctx = [int(c) for c in inputs["ctx_lens"]]
    if w.ctx_range:
        ctxs = f"ctx {min(ctx)}..{max(ctx)} (uniform {w.ctx_range[0]}..{w.ctx_range[1]}, mean {np.mean(ctx):.0f})"
    else:
        ctxs = f"ctx {w.ctx} ({w.image} image + {w.ctx - w.image} text) per sequence"
    dt = "bf16" if w.dtype == "bf16" else "fp32"
    parts = [f"{w.name}: batch {w.batch}, {w.hq}/{w.hkv} heads, head_dim {w.d}, {dt}, {ctxs}"]
    if "draft" in w.steps:
        parts.append(f"draft block {w.n_draft}")
    if "verify" in w.steps or "accept" in w.steps:
        parts.append(f"tree {w.n_tree} rows")
    if "accept" in w.steps:
        parts.append(f"vocab {w.vocab}")
    return ", ".join(parts) + "; steps: " + " + ".join(w.steps)


def measure_config(args, name, G, C, torch, np, dev, stream, headline):
    w = C.WORKLOADS[name]
    t_gen = time.perf_counter()
    inputs, sets = prepare_sets(w, args.sets, G, C, torch, dev)
    t_gen = time.perf_counter() - t_gen
    torch.cuda.synchronize()
    rt = time_rounds(args, sets, stream, torch, np)
    k_us, c_us = kernel_times(args, sets, stream, G, torch, np)
    work, kvb = round_work(w, inputs)
    per_kernel = per_kernel_report(w, work, k_us, c_us)
    us_round = rt["wall_us"]
    res = {
        "metric": HEADLINE_METRIC if headline else f"round latency (\u00b5s) of the {name} configuration, 1 MI355X",
        "value": round(us_round, 2),
        "unit": "us per round",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(us_round / 1e3, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": describe(w, inputs), "global_batch": w.batch,
                   "seq_len": int(max(int(c) for c in inputs["ctx_lens"])), "parallelism": "single GPU",
                   "launch": rt["launch"], "input_sets_rotated": args.sets},
        "round_us_p10_p50_p90": {"cold": rt["cold"], "warm": rt["warm"]},
        "kernels": per_kernel,
        "input_gen_s": round(t_gen, 1),
    }
    if "draft" in k_us or "verify" in k_us:
        att = [k for k in ("draft", "verify") if k in k_us]
        res["achieved_kv_gbps"] = round(len(att) * kvb / sum(k_us[k] for k in att) / 1e3, 1)
        # the same with each attention call's merge pass (whole call time)
        res["achieved_kv_gbps_with_merge"] = round(len(att) * kvb / sum(c_us[k] for k in att) / 1e3, 1)
        res["round_kv_gbps"] = round(len(att) * kvb / us_round / 1e3, 1)
    return w, inputs, sets, res, k_us, c_us, work


def roofline(w, k_us, c_us, work, per_kernel):
    dom = max(k_us, key=lambda k: k_us[k])
    if dom == "verify" and w.dtype == "bf16":
        ach = work["verify"]["flops"] / k_us["verify"] / 1e6
        roof = {"bound": "mfma", "achieved": round(ach, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s"}
    else:
        ach = work[dom]["bytes"] / k_us[dom] / 1e3
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    # the dominant step as the whole call (attention + its merge pass)
    roof["frac_with_merge"] = round(roof["frac"] * k_us[dom] / c_us[dom], 4)
    src = os.path.join(ROOT, "paper_2609_00355_amd", "csrc",
                       "accept.hip" if dom == "accept" else "attn_bf16.hip" if w.dtype == "bf16" else "attn_f32.hip")
    roof["traffic"] = load_traffic(dom, src, w.name)
    roof["kernel"] = per_kernel[dom]["kernel"]
    roof["launch_us"] = round(k_us[dom], 2)
    return roof


def main():
    args = parse()
    if args.traffic_from:
        summarise_traffic(*args.traffic_from, args.workload)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path (asked for --gpus {args.gpus}, "
              f"WORLD_SIZE={world}). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2609_00355_amd as G
    from workloads import configs as C

    if not os.path.exists(G.LIB_PATH):
        from paper_2609_00355_amd import build
        build.build()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")

    if args.verify_sweep:
        verify_sweep(args, C.WORKLOADS[args.workload], G, C, torch, np, dev)
        return

    # the prepared calls are bound to this stream; graphs are captured on it
    stream = torch.cuda.Stream()
    torch.cuda.set_stream(stream)

    for name in [c for c in args.configs.split(",") if c and c != args.workload]:
        w, inputs, sets, res, k_us, c_us, work = measure_config(args, name, G, C, torch, np, dev, stream,
                                                                headline=False)
        res["roofline"] = roofline(w, k_us, c_us, work, res["kernels"])
        if not args.no_cpu_baseline:
            res["cpu_baseline"] = cpu_baseline(inputs, args.cpu_seconds_config)
        print(json.dumps(res), flush=True)
        del sets, inputs
        torch.cuda.empty_cache()

    w, inputs, sets, res, k_us, c_us, work = measure_config(args, args.workload, G, C, torch, np, dev, stream,
                                                            headline=True)
    if args.calibrate_copy:  # reference kernel for the HBM byte counters
        src_c = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
        dst_c = torch.empty_like(src_c)
        for _ in range(3):
            torch.neg(src_c, out=dst_c)  # a plain streaming kernel: reads and writes COPY_BYTES
        torch.cuda.synchronize()
        del src_c, dst_c
    res["roofline"] = roofline(w, k_us, c_us, work, res["kernels"])
    if not args.eager and w.steps == ("draft", "verify", "accept"):
        eager_args = argparse.Namespace(**{**vars(args), "eager": True})
        res["eager_round_us"] = round(time_rounds(eager_args, sets, stream, torch, np)["wall_us"], 2)
    if w.steps == ("draft", "verify", "accept") and w.dtype == "bf16":
        acc = sets[0]["a_out"]["accept_len"].cpu().numpy()
        res["synthetic_tau"] = round(1.0 + float(acc.mean()), 3)
        if not args.no_tree:
            res["tree_builder"] = measure_tree_builder(args, w, G, C, torch, np, dev, stream)
        res["commit"] = measure_commit(args, w, sets[0], G, torch, np, dev, stream, inputs["ctx_lens"])
        res["sample_accept"] = measure_sample(args, w, sets, G, torch, np, stream)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(inputs, args.cpu_seconds)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
