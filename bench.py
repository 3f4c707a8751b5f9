#!/usr/bin/env python3
"""Throughput of one context-parallel rank's share of FlashCP's attention
(forward + backward) on one MI355X.

A step is the whole path once over one synthetic packed sequence: the shard
plan and rank view (host, C++), the table upload, the KV gather that stands
in for the sharding-aware receive, the local and received forward partial
passes and their log-sum-exp merge (one launch: each workgroup merges its
query tile's two partials in its epilogue), the backward preprocess, and
the key-major dK/dV and query-major dQ passes.
Inputs are resident in HBM before timing starts. The metric counts useful
FLOPs: 14 * d * Hq * pairs, pairs being the visible (query, key) pairs per
head of the rank (sum of its shards' W_i); masked lanes never count.

Prints one JSON line. Only one GPU is supported.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "useful attention TFLOP/s (fwd+bwd) per CP-rank shard; % of bf16 MFMA peak"
BF16_PEAK_TFLOPS = 2516.6   # 256 CUs x 2.4 GHz x 4096 bf16 flop/clk/CU (dense)
HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama8b")
    ap.add_argument("--mode", choices=["two_pass"], default="two_pass")
    ap.add_argument("--bwd", choices=["det", "atomic"], default="det",
                    help="backward mode: deterministic (query-major dQ pass) or atomic "
                         "(dQ added by the key-major pass)")
    ap.add_argument("--delta-from", choices=["f32", "bf16"], default="f32",
                    help="output the backward preprocess reads: the forward's fp32 O (also "
                         "written by the forward) or its bf16 O")
    ap.add_argument("--bm-fwd", type=int, default=0,
                    help="forward / dQ query tile rows (32, 64, 128; 0: the view's default)")
    ap.add_argument("--workloads", type=int, default=1,
                    help="also time the other workloads (GPU legs only) into the 'workloads' key")
    ap.add_argument("--workload-steps", type=int, default=10,
                    help="timed steps of each other workload")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="budget of the CPU-oracle baseline sample (0 disables it)")
    ap.add_argument("--study", choices=["planner", "granularity", "tiles"], default=None,
                    help="instead of the step benchmark: the planner-quality study (host "
                         "only), the shard-granularity kernel study, or the forward tile-shape "
                         "sweep; JSON lines, then a table")
    ap.add_argument("--seeds", type=int, default=5, help="length seeds per planner-study row")
    return ap.parse_args()


# ------------------------------------------------------------------ studies

PLANNERS = ["per_seq", "per_doc", "whole_lpt", "hybrid"]


def run_planner(F, name, cu, cp):
    if name == "per_seq":
        return F.fc_plan_per_seq(cu, cp)
    if name == "per_doc":
        return F.fc_plan_per_doc(cu, cp)
    if name == "whole_lpt":
        return F.fc_plan_whole_lpt(cu, cp)
    return F.fc_plan_hybrid(cu, cp)[0]


def brute_whole_doc(F, cu, cp):
    """Least max-workload over every whole-document placement (cp**n of
    them; small cases only), the optimum the ILP of Sec. 3.4 would find
    among whole-document plans."""
    import itertools
    n = len(cu) - 1
    best = None
    for assign in itertools.product(range(cp), repeat=n):
        if assign[0] != 0:   # worker relabelling: fix document 0 on worker 0
            continue
        plan = np.array([[k, assign[k], 0, int(cu[k + 1] - cu[k])] for k in range(n)], dtype=np.int32)
        w = max(F.fc_plan_stats(cu, cp, plan, 1, 1)["work"])
        best = w if best is None else min(best, w)
    return best


def study_planner(args):
    """Planner quality on synthetic lengths (a host-only analogue of the
    paper's Table 2 without its datasets or ILP solver): imbalance max W /
    mean W, token spread, received-KV tokens |R_r| (max over workers), the
    Eq. 4 and Eq. 5 volumes, and the C++ planner's time per sequence; plus,
    on small cases, each planner's max W against the best whole-document
    placement found by brute force."""
    from paper_2606_08476_amd import flashcp as F
    from paper_2606_08476_amd import synth
    rows = []
    sweeps = [("llama8b", cp) for cp in (2, 4, 8, 16, 32)] + [("wholedoc", 8), ("longdoc", 16),
                                                              ("hybrid70b", 32)]
    for wl, cp in sweeps:
        w = synth.WORKLOADS[wl]
        acc = {p: {"imbalance": [], "tok_spread": [], "recv_max": [], "eq4": [], "eq5": [],
                   "ms": []} for p in PLANNERS}
        for seed in range(args.seeds):
            cu = synth.cu_seqlens(synth.doc_lengths(wl, seed=100 + seed))
            for pn in PLANNERS:
                t = []
                for _ in range(3):
                    t0 = time.perf_counter()
                    plan = run_planner(F, pn, cu, cp)
                    t.append(time.perf_counter() - t0)
                st = F.fc_plan_stats(cu, cp, plan, w.hkv, w.d)
                a = acc[pn]
                a["imbalance"].append(st["imbalance"])
                a["tok_spread"].append(max(st["tokens"]) / (sum(st["tokens"]) / cp))
                a["recv_max"].append(max(st["recv_tokens"]))
                a["eq4"].append(st["eq4"])
                a["eq5"].append(st["eq5"])
                a["ms"].append(sorted(t)[1] * 1e3)
        for pn in PLANNERS:
            a = acc[pn]
            row = {"study": "planner", "workload": wl, "context": w.context, "cp": cp, "planner": pn,
                   "seeds": args.seeds,
                   "imbalance_mean": round(float(np.mean(a["imbalance"])), 4),
                   "imbalance_max": round(float(np.max(a["imbalance"])), 4),
                   "max_tokens_over_mean": round(float(np.mean(a["tok_spread"])), 4),
                   "recv_tokens_max": int(np.mean(a["recv_max"])),
                   "eq4_elems": int(np.mean(a["eq4"])), "eq5_elems": int(np.mean(a["eq5"])),
                   "planner_ms": round(float(np.median(a["ms"])), 3)}
            rows.append(row)
            print(json.dumps(row), flush=True)
    # small cases: against the best whole-document placement
    rng = np.random.default_rng(11)
    small = []
    for cp, nd in ((2, 8), (2, 10), (3, 7), (4, 7)):
        ratios = {p: [] for p in PLANNERS}
        for _ in range(args.seeds):
            lens = [int(x) for x in np.exp(rng.normal(np.log(512), 1.0, size=nd)).clip(16, 8192)]
            lens[-1] += (-sum(lens)) % cp
            cu = synth.cu_seqlens(np.array(lens))
            opt = brute_whole_doc(F, cu, cp)
            for pn in PLANNERS:
                w_max = max(F.fc_plan_stats(cu, cp, run_planner(F, pn, cu, cp), 1, 1)["work"])
                ratios[pn].append(w_max / opt)
        row = {"study": "planner_vs_brute_force", "cp": cp, "docs": nd, "seeds": args.seeds,
               **{f"{p}_maxW_over_best_whole_doc": round(float(np.mean(r)), 4) for p, r in ratios.items()}}
        small.append(row)
        print(json.dumps(row), flush=True)
    print("\n| lengths | N | planner | imbalance (mean / max) | max tokens / mean | max recv tokens | Eq. 4 | Eq. 5 | planner ms |")
    print("|---|---|---|---|---|---|---|---|---|")
    for r in rows:
        print(f"| {r['workload']} ({r['context']}) | {r['cp']} | {r['planner']} | {r['imbalance_mean']} / "
              f"{r['imbalance_max']} | {r['max_tokens_over_mean']} | {r['recv_tokens_max']} | "
              f"{r['eq4_elems']:.3g} | {r['eq5_elems']:.3g} | {r['planner_ms']} |")
    print("\n| N | docs | " + " | ".join(PLANNERS) + " |")
    print("|---|---|" + "---|" * len(PLANNERS))
    for r in small:
        print(f"| {r['cp']} | {r['docs']} | " + " | ".join(
            str(r[f'{p}_maxW_over_best_whole_doc']) for p in PLANNERS) + " |")


def plan_for(F, w, cu):
    if w.plan == "per_doc":
        return F.fc_plan_per_doc(cu, w.cp)
    if w.plan == "whole_lpt":
        return F.fc_plan_whole_lpt(cu, w.cp)
    return F.fc_plan_hybrid(cu, w.cp)[0]


def rank_for(F, w, cu, plan):
    if w.rank == "last":
        return w.cp - 1
    if w.rank == "heaviest":
        work = F.fc_plan_stats(cu, w.cp, plan, w.hkv, w.d)["work"]
        return int(np.argmax(work))
    return int(w.rank)


def measured_traffic(entry, workload):
    """HBM bytes per launch of a kernel from the committed counter summaries
    (profiles/traffic_*.md, FETCH_SIZE and WRITE_SIZE scaled by a copy
    kernel of known size); None when there is no record for this kernel and
    workload, or when the kernel's sources changed since it was taken."""
    import glob
    import hashlib
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "traffic_*.md"))):
        for line in open(path):
            if not line.startswith("traffic-record:"):
                continue
            rec = json.loads(line.split(":", 1)[1])
            if rec.get("entry") != entry or rec.get("workload") != workload:
                continue
            h = hashlib.sha256()
            for src in rec["sources"]:
                with open(os.path.join(ROOT, src), "rb") as f:
                    h.update(f.read())
            if h.hexdigest() != rec["sources_sha256"]:
                return None
            return int(rec["fetch_bytes_per_launch"]) + int(rec["write_bytes_per_launch"])
    return None


def cpu_baseline(cu, view_tables, x, w, seconds):
    """The oracle (fp32, as it stands) on whole document segments of the
    rank, forward + backward, until the time budget is used."""
    import torch
    from oracle import attention as A
    qg, rg = view_tables["q_gpos"].astype(np.int64), view_tables["recv_gpos"].astype(np.int64)
    qcu = view_tables["q_cu_docseg"]
    rcu = view_tables["recv_cu"]
    kv = np.concatenate([qg, rg])
    k = torch.cat([x["k_loc"], x["k_recv"]])
    v = torch.cat([x["v_loc"], x["v_recv"]])
    torch.set_num_threads(max(1, min(os.cpu_count() or 1, int(os.environ.get("OMP_NUM_THREADS", "16")))))
    # smallest segments first, so the sample finishes within the budget
    segs = sorted(range(len(qcu) - 1), key=lambda s: int(qcu[s + 1] - qcu[s]) * int(rcu[s + 1] - rcu[s] + qcu[s + 1] - qcu[s]))
    pairs = 0
    done = 0
    t0 = time.perf_counter()
    for s in segs:
        rows = np.arange(qcu[s], qcu[s + 1])
        A.attention_fwd(cu, qg, x["q"], kv, k, v, rows=rows, dtype=torch.float32)
        A.attention_bwd(cu, qg, x["q"], kv, k, v, x["do"], rows=rows, dtype=torch.float32)
        n = int(rows.size)
        # pairs of this segment: local causal + received prefix per row
        lim = view_tables["lim"][rows] - rcu[s]
        pairs += n * (n + 1) // 2 + int(lim.sum())
        done += 1
        if time.perf_counter() - t0 >= seconds:
            break
    dt = time.perf_counter() - t0
    flops = 14.0 * w.d * w.hq * pairs
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": torch.get_num_threads(),
            "kind": "oracle",
            "sample": f"{done} of {len(segs)} document segments of the same rank share (smallest first), "
                      f"{pairs} pairs/head = {100.0 * pairs / max(1, view_tables['pairs']):.2f}% of the "
                      f"rank's work, forward + backward in fp32, {dt:.1f} s"}


def study_granularity(args):
    """Kernel efficiency against shard granularity on one GPU (an analogue of
    the paper's kernel-efficiency figure, Sec. 2.3): one 128K-token document
    and 16 documents of 8K, each run unsharded (one rank holds every query)
    and as every rank's share under Per-Doc and per-sequence (Llama3 CP)
    plans at N = 4 and 8. Each configuration runs all of its ranks' shares
    one after another (gather, forward partials, merge, backward) and
    reports useful TFLOP/s over the summed time, and over N times the
    slowest rank (the step time of an N-GPU run with a free exchange)."""
    import torch
    from paper_2606_08476_amd import flashcp as F
    from paper_2606_08476_amd import synth
    dev = torch.device("cuda:0")
    hq, hkv, d = 32, 8, 128
    bf, f32 = torch.bfloat16, torch.float32
    patterns = {"1x128K": [131072], "16x8K": [8192] * 16}
    configs = [("whole", 1), ("per_doc", 4), ("per_doc", 8), ("per_seq", 4), ("per_seq", 8)]
    rows = []
    g = torch.Generator(device=dev)
    for pname, lens in patterns.items():
        cu = synth.cu_seqlens(np.array(lens))
        T = int(cu[-1])
        g.manual_seed(7)
        q_all = torch.randn(T, hq, d, device=dev, generator=g).to(bf)
        do_all = torch.randn(T, hq, d, device=dev, generator=g).to(bf)
        k_pk = torch.randn(T, hkv, d, device=dev, generator=g).to(bf)
        v_pk = torch.randn(T, hkv, d, device=dev, generator=g).to(bf)
        for kind, cp in configs:
            plan = F.fc_plan_whole_lpt(cu, 1) if kind == "whole" else run_planner(F, kind, cu, cp)
            per_rank = []
            pairs_total = 0
            for rank in range(cp):
                v = F.View(cu, plan, cp, rank, hq, hkv, d).bind(dev)
                i = v.info
                tq, tr = i["t_q"], i["t_recv"]
                pairs_total += i["pairs_loc"] + i["pairs_recv"]
                qg = torch.from_numpy(v.export()["q_gpos"].astype(np.int64)).to(dev)
                q, do = q_all[qg].contiguous(), do_all[qg].contiguous()
                e = lambda *sh, dt=f32: torch.empty(*sh, dtype=dt, device=dev)
                kl, vl = e(tq, hkv, d, dt=bf), e(tq, hkv, d, dt=bf)
                kr, vr = e(tr, hkv, d, dt=bf), e(tr, hkv, d, dt=bf)
                o, lse, delta = e(tq, hq, d, dt=bf), e(hq, tq), e(hq, tq)
                o32 = e(tq, hq, d)
                dq, dkl, dvl = e(tq, hq, d), e(tq, hkv, d), e(tq, hkv, d)
                dkr, dvr = e(tr, hkv, d), e(tr, hkv, d)
                ws = torch.empty(max(v.workspace_size()[2], 1), dtype=torch.uint8, device=dev)
                fws = torch.empty(max(v.workspace_size(F.FC_TWO_PASS)[0], 1), dtype=torch.uint8,
                                  device=dev)

                def run():
                    F.fc_kv_gather(v, k_pk, v_pk, kl, vl, kr, vr)
                    F.fc_attn_fwd(v, q, kl, vl, kr, vr, 0.0, F.FC_TWO_PASS, o, o32, lse, fws)
                    F.fc_bwd_preprocess(v, o, do, delta, o_f32=o32)
                    F.fc_attn_bwd_pass(v, q, kl, vl, kr, vr, lse, delta, do, 0.0, dq, dkl, dvl, dkr, dvr, ws)

                for _ in range(2):
                    run()
                torch.cuda.synchronize()
                ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
                reps = 5
                ev[0].record()
                for _ in range(reps):
                    run()
                ev[1].record()
                torch.cuda.synchronize()
                per_rank.append(ev[0].elapsed_time(ev[1]) / reps)
                v.close()
            flops = 14.0 * d * hq * pairs_total
            tsum, tmax = sum(per_rank), max(per_rank)
            row = {"study": "granularity", "pattern": pname, "plan": kind, "cp": cp,
                   "pairs_per_head": int(pairs_total),
                   "sum_ms": round(tsum, 3), "max_rank_ms": round(tmax, 3),
                   "tflops_sum": round(flops / (tsum * 1e-3) / 1e12, 1),
                   "tflops_n_x_max": round(flops / (cp * tmax * 1e-3) / 1e12, 1)}
            rows.append(row)
            print(json.dumps(row), flush=True)
    print("\n| documents | plan | N | pairs/head | sum over ranks ms | slowest rank ms | TFLOP/s (sum) | TFLOP/s (N x slowest) |")
    print("|---|---|---|---|---|---|---|---|")
    for r in rows:
        print(f"| {r['pattern']} | {r['plan']} | {r['cp']} | {r['pairs_per_head']:.4g} | {r['sum_ms']} | "
              f"{r['max_rank_ms']} | {r['tflops_sum']} | {r['tflops_n_x_max']} |")


def measure(args, name, steps, warmup, dev):
    """The timed step on one workload: plan, view, gather, two-pass forward,
    preprocess, backward pass; per-kernel times from HIP events on the
    step's stream, the step from the host clock around `steps` steps."""
    import torch
    from paper_2606_08476_amd import flashcp as F
    from paper_2606_08476_amd import synth

    w = synth.WORKLOADS[name]
    lens = synth.doc_lengths(name)
    cu = synth.cu_seqlens(lens)
    plan = plan_for(F, w, cu)
    rank = rank_for(F, w, cu, plan)
    tiles = (args.bm_fwd, 0, 0, 0)
    view = F.View(cu, plan, w.cp, rank, w.hq, w.hkv, w.d, tiles=tiles)
    info = view.info
    tab = view.export()
    tq, tr, hq, hkv, d = info["t_q"], info["t_recv"], w.hq, w.hkv, w.d
    pairs = info["pairs_loc"] + info["pairs_recv"]
    tab["pairs"] = pairs

    # inputs, resident in HBM before timing
    src = synth.TensorSource(w.index, hq, hkv, d)
    qg, rg = tab["q_gpos"], tab["recv_gpos"]
    x = {"q": src.rows("q", qg), "do": src.rows("do", qg), "k_loc": src.rows("k", qg),
         "v_loc": src.rows("v", qg), "k_recv": src.rows("k", rg), "v_recv": src.rows("v", rg)}
    T = int(cu[-1])
    bf, f32 = torch.bfloat16, torch.float32
    k_pk = torch.zeros(T, hkv, d, dtype=bf, device=dev)
    v_pk = torch.zeros(T, hkv, d, dtype=bf, device=dev)
    k_pk[torch.from_numpy(qg.astype(np.int64)).to(dev)] = x["k_loc"].to(dev)
    v_pk[torch.from_numpy(qg.astype(np.int64)).to(dev)] = x["v_loc"].to(dev)
    if tr:
        k_pk[torch.from_numpy(rg.astype(np.int64)).to(dev)] = x["k_recv"].to(dev)
        v_pk[torch.from_numpy(rg.astype(np.int64)).to(dev)] = x["v_recv"].to(dev)
    q = x["q"].to(dev)
    do = x["do"].to(dev)
    k_loc = torch.empty(tq, hkv, d, dtype=bf, device=dev)
    v_loc = torch.empty_like(k_loc)
    k_recv = torch.empty(tr, hkv, d, dtype=bf, device=dev)
    v_recv = torch.empty_like(k_recv)
    o = torch.empty(tq, hq, d, dtype=bf, device=dev)
    o32 = torch.empty(tq, hq, d, dtype=f32, device=dev) if args.delta_from == "f32" else None
    lse = torch.empty(hq, tq, dtype=f32, device=dev)
    delta = torch.empty(hq, tq, dtype=f32, device=dev)
    dq = torch.empty(tq, hq, d, dtype=f32, device=dev)
    dk_loc = torch.empty(tq, hkv, d, dtype=f32, device=dev)
    dv_loc = torch.empty_like(dk_loc)
    dk_recv = torch.empty(tr, hkv, d, dtype=f32, device=dev)
    dv_recv = torch.empty_like(dk_recv)
    meta = torch.empty(int(info["meta_bytes"]) + 256, dtype=torch.uint8, device=dev)
    fwd_ws = torch.empty(max(view.workspace_size(F.FC_TWO_PASS)[0], 1), dtype=torch.uint8, device=dev)
    dkdv_ws = torch.empty(view.workspace_size()[2], dtype=torch.uint8, device=dev)
    names = ["kv_gather", "attn_fwd", "bwd_preprocess", "attn_bwd"]
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)]
    acc = np.zeros(len(names))
    kept = []

    def step():
        p = plan_for(F, w, cu)
        v = F.View(cu, p, w.cp, rank, hq, hkv, d, tiles=tiles).bind(dev, meta)
        kept.append(v)
        ev[0].record()
        F.fc_kv_gather(v, k_pk, v_pk, k_loc, v_loc, k_recv, v_recv)
        ev[1].record()
        # both partial passes (received keys, then local keys) and their
        # log-sum-exp merge in one launch; with no received KV the local pass
        # alone writes the final O and LSE
        F.fc_attn_fwd(v, q, k_loc, v_loc, k_recv, v_recv, 0.0, F.FC_TWO_PASS, o, o32, lse, fwd_ws)
        ev[2].record()
        # delta = rowsum(dO * O) from the fp32 O (exact to fp32; from the bf16
        # O its rounding reaches every dS of the row)
        F.fc_bwd_preprocess(v, o, do, delta, o_f32=o32)
        ev[3].record()
        # dK/dV (key-major) and dQ (query-major) workgroups in one launch
        F.fc_attn_bwd_pass(v, q, k_loc, v_loc, k_recv, v_recv, lse, delta, do, 0.0, dq, dk_loc,
                           dv_loc, dk_recv, dv_recv, dkdv_ws, deterministic=args.bwd == "det")
        ev[4].record()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    kept.clear()
    t0 = time.perf_counter()
    per = []
    for _ in range(steps):
        step()
        # per-kernel durations are read after the loop from stored copies
        per.append([ev[i] for i in range(len(ev))])
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)]
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    for e in per:
        for i in range(len(names)):
            acc[i] += e[i].elapsed_time(e[i + 1])
    acc /= steps
    # the merge kernel alone (outside the timed steps): the step merges in the
    # forward's epilogue, this is fc_lse_merge for partials made apart
    merge_side = None
    if tr:
        o_a, o_b = (torch.empty(tq, hq, d, dtype=f32, device=dev) for _ in range(2))
        l_a, l_b = (torch.empty(hq, tq, dtype=f32, device=dev) for _ in range(2))
        F.fc_attn_fwd_partials(kept[-1], q, k_loc, v_loc, k_recv, v_recv, 0.0, o_a, l_a, o_b, l_b)
        me = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        for _ in range(3):
            F.fc_lse_merge(o_a, l_a, o_b, l_b, o, None, lse)
        me[0].record()
        for _ in range(20):
            F.fc_lse_merge(o_a, l_a, o_b, l_b, o, None, lse)
        me[1].record()
        torch.cuda.synchronize()
        mms = me[0].elapsed_time(me[1]) / 20
        gbs = tq * hq * (2 * 4 * d + 2 * 4 + 2 * d + 4) / (mms * 1e-3) / 1e9
        merge_side = {"ms": round(mms, 4), "gbs": round(gbs, 1),
                      "frac_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
                      "note": "fc_lse_merge alone, not in the step (the step merges in the forward)"}
        del o_a, o_b, l_a, l_b

    for v in kept:
        v.close()
    kept.clear()
    view.close()

    ms = wall * 1e3 / steps
    useful = 14.0 * d * hq * pairs
    value = useful / (ms * 1e-3) / 1e12
    # per-kernel algorithmic work
    kv_rows = tq + tr
    work = {
        "kv_gather": ("hbm", 2 * 2 * kv_rows * hkv * d * 2),
        # both partial passes (4d per pair) with the merge in their epilogue
        "attn_fwd": ("mfma", 4.0 * d * hq * pairs),
        # dO (bf16) and O (fp32, or bf16) read, delta written
        "bwd_preprocess": ("hbm", tq * hq * (2 * d + (4 if o32 is not None else 2) * d + 4)),
        # backward, algorithmic: S recomputed once, dP, dV, dK, dQ (10d per
        # pair, the FlashAttention count); the deterministic kernels execute
        # 14d (the dQ workgroups recompute S and dP), reported apart as
        # executed_tflops
        "attn_bwd": ("mfma", 10.0 * d * hq * pairs),
    }
    executed = {"attn_bwd": (14.0 if args.bwd == "det" else 10.0) * d * hq * pairs}
    kernels = {}
    for i, n in enumerate(names):
        kind, amount = work[n]
        t = acc[i] * 1e-3
        if amount == 0 or acc[i] <= 0:
            kernels[n] = {"ms": round(acc[i], 4)}
            continue
        if kind == "mfma":
            a = amount / t / 1e12
            kernels[n] = {"ms": round(acc[i], 4), "tflops": round(a, 1), "frac_bf16_peak": round(a / BF16_PEAK_TFLOPS, 4)}
            if n in executed:
                kernels[n]["executed_tflops"] = round(executed[n] / t / 1e12, 1)
        else:
            a = amount / t / 1e9
            kernels[n] = {"ms": round(acc[i], 4), "gbs": round(a, 1), "frac_hbm_peak": round(a / HBM_PEAK_GBS, 4)}
    dom = max(range(len(names)), key=lambda i: acc[i])
    dn = names[dom]
    kind, amount = work[dn]
    traffic = measured_traffic(dn, w.name)
    if kind == "mfma":
        ach = amount / (acc[dom] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 2), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(ach / BF16_PEAK_TFLOPS, 4), "traffic": traffic, "kernel": dn}
    else:
        ach = amount / (acc[dom] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": traffic, "kernel": dn}
    return dict(w=w, rank=rank, cu=cu, tab=tab, x=x, tq=tq, tr=tr, pairs=pairs, useful=useful,
                bm_fwd=info["bm_fwd"],
                ms=ms, value=value, kernels=kernels, roof=roof, merge_side=merge_side,
                steps=steps, warmup=warmup)


def study_tiles(args):
    """Forward / dQ query-tile shape against step time on every workload:
    bm_fwd = 32, 64, 128 rows (4, 2, 1 query heads of a KV group per
    workgroup; the shapes the group size allows), the step timed as in the
    benchmark."""
    import torch
    from paper_2606_08476_amd import synth
    dev = torch.device("cuda:0")
    rows = []
    for name, w in synth.WORKLOADS.items():
        G = w.hq // w.hkv
        for bm in (32, 64, 128):
            if G % (128 // bm):
                continue
            args.bm_fwd = bm
            m = measure(args, name, args.workload_steps, 2, dev)
            k = m["kernels"]
            row = {"study": "tiles", "workload": name, "bm_fwd": bm, "ms_per_step": round(m["ms"], 4),
                   "tflops": round(m["value"], 1), "fwd_ms": k["attn_fwd"]["ms"],
                   "bwd_ms": k["attn_bwd"]["ms"]}
            rows.append(row)
            print(json.dumps(row), flush=True)
            del m
            torch.cuda.empty_cache()
    print("\n| workload | bm_fwd | step ms | TFLOP/s | forward ms | backward ms |")
    print("|---|---|---|---|---|---|")
    for r in rows:
        print(f"| {r['workload']} | {r['bm_fwd']} | {r['ms_per_step']} | {r['tflops']} | "
              f"{r['fwd_ms']} | {r['bwd_ms']} |")


def describe(m):
    w = m["w"]
    return (f"{w.name}: {w.context}-token packed context, CP degree {w.cp}, {w.plan} plan, "
            f"rank {m['rank']}; {w.hq} query / {w.hkv} KV heads, d {w.d}")


def main():
    args = parse()
    if args.study == "planner":
        study_planner(args)
        return
    if args.study == "granularity":
        study_granularity(args)
        return
    if args.study == "tiles":
        study_tiles(args)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this build runs one rank's share on one GPU; --gpus must be 1 "
              "(multi-GPU exchange is not part of it)", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2606_08476_amd import synth

    dev = torch.device("cuda:0")
    m = measure(args, args.workload, args.steps, args.warmup, dev)
    w, d, hq = m["w"], m["w"].d, m["w"].hq
    ms, value = m["ms"], m["value"]
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": describe(m) + "; two-pass forward (received and local partials and "
                               "their LSE merge in one launch), key-major dK/dV and query-major dQ "
                               "backward" + ("" if args.bwd == "det" else " (dQ by atomics)"),
                   "t_q": m["tq"], "t_recv": m["tr"], "pairs_per_head": m["pairs"],
                   "useful_tflop_per_step": round(m["useful"] / 1e12, 4),
                   "pct_of_bf16_peak": round(100 * value / BF16_PEAK_TFLOPS, 2),
                   "strict_tflops_12d": round(12.0 * d * hq * m["pairs"] / (ms * 1e-3) / 1e12, 2),
                   "bwd_mode": "deterministic" if args.bwd == "det" else "atomic dQ",
                   "bm_fwd": m["bm_fwd"],
                   "delta_from": "fp32 O" if args.delta_from == "f32" else "bf16 O"},
        "roofline": m["roof"],
        "kernels": m["kernels"],
        "lse_merge_alone": m["merge_side"],
    }
    # the other workloads, GPU legs only, after the headline one
    if args.workloads:
        wl = {}
        for name in synth.WORKLOADS:
            r = m if name == args.workload else measure(args, name, args.workload_steps, 2, dev)
            wl[name] = {
                "config": describe(r), "t_q": r["tq"], "t_recv": r["tr"], "pairs_per_head": r["pairs"],
                "bm_fwd": r["bm_fwd"],
                "steps": r["steps"], "ms_per_step": round(r["ms"], 4), "tflops": round(r["value"], 2),
                "pct_of_bf16_peak": round(100 * r["value"] / BF16_PEAK_TFLOPS, 2),
                "kernels": r["kernels"], "roofline_kernel": r["roof"]["kernel"],
                "roofline_frac": r["roof"]["frac"],
                "lse_merge_alone_gbs": r["merge_side"]["gbs"] if r["merge_side"] else None}
            if r is not m:
                del r
                torch.cuda.empty_cache()
        out["workloads"] = wl
    if args.cpu_seconds > 0:
        out["cpu_baseline"] = cpu_baseline(m["cu"], m["tab"], m["x"], w, args.cpu_seconds)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
