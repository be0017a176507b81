"""Benchmark: one step = one full validation pass of the combined cross-layer
workload (selector evaluation, flow tracing, masked reachability, per-intent
verdict) on one GPU, inputs resident in HBM.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload cfg5|small]

Prints one JSON line.  `value` is selector evaluations ((intent, node)
pairs) per second of whole-step time; flow lookups ("hops traced") per
second of whole-step time are reported beside it, with per-kernel times,
the roofline of the dominant kernel, and the CPU oracle timed on a bounded
sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# VALU issue peak: two wave-wide 32-bit instructions per CU per clock (256 CUs x
# 128 lanes x 2.4 GHz = 78.6 T lane-ops/s, the rate the published 157.3 TFLOP/s
# fp32 vector peak implies at two flops per lane-op).  pc_measure_valu reaches
# 0.93-0.96 of it with two-source 32-bit operations on vector registers and
# constants; an operation with a scalar-register operand, a third source or a
# 64-bit operand issues at half of it (measured 0.48-0.50).
VALU_PEAK_LANE_OPS = 256 * 128 * 2.4e9
# scalar ALU: one instruction per CU per clock (measured 0.96 of it)
SALU_PEAK_INSTR = 256 * 2.4e9

# HBM bytes per launch of k_sel_eval, k_aff_eval and k_tr_prep (per step of
# k_tr_match) on the combined workload, from one rocprofv3 FETCH_SIZE pass and
# one WRITE_SIZE pass each, scaled by what the same counter reads for a plain
# copy of known size (the command lines and counter values are in
# profiles/k_sel_eval_k_tr_prep_cfg5_hbm_counters.md).  Valid only for the
# kernel source they were measured on.
TRAFFIC = [
    {"source": "paper_2602_16100_amd/csrc/select.hip",
     "sha256": "3ba266f186a97c69f5525e79cbd1aa8e8de7774ba0177ee4f0f28a75ebc43f74",
     "workload": "cfg5",
     "bytes_per_launch": {"k_sel_eval": 680_687_937 + 4_407_406_605,
                          "k_aff_eval": 1_360_481_846 + 4_407_121_613}},
    {"source": "paper_2602_16100_amd/csrc/trace.hip",
     "sha256": "c9b11ae36f815781b39e2ccddb1fca6cd58dc757cfef139cb8fdfc38042cac7d",
     "workload": "cfg5",
     # k_tr_match: per step (its 6 launches), like the hop-loop roofline
     "bytes_per_launch": {"k_tr_prep": 1_888_686_134 + 566_231_040,
                          "k_tr_match": 2_325_285_696 + 142_260_102}},
    # the single-kernel configurations (profiles/cfg2_cfg3_cfg4_hbm_counters.md)
    {"source": "paper_2602_16100_amd/csrc/select.hip",
     "sha256": "3ba266f186a97c69f5525e79cbd1aa8e8de7774ba0177ee4f0f28a75ebc43f74",
     "workload": "cfg2",
     "bytes_per_launch": {"k_sel_eval": 61_279_026 + 206_234_144}},
    {"source": "paper_2602_16100_amd/csrc/trace.hip",
     "sha256": "c9b11ae36f815781b39e2ccddb1fca6cd58dc757cfef139cb8fdfc38042cac7d",
     "workload": "cfg3-rpath",
     "bytes_per_launch": {"k_tr_match": 1_056_617_428 + 793_564_755}},  # per call (its 7 launches)
    {"source": "paper_2602_16100_amd/csrc/reach.hip",
     "sha256": "c5686db7947fd48ea645f261a5cf397dcff66e0567c993962d5520fdb59c8dee",
     "workload": "cfg4",
     # per call: k_rc_validate, the -1 fill and k_rc_queue
     "bytes_per_launch": {"pc_masked_reach": 47_662_753 + 1_047_437_664}},
]


# Issue counters of k_tr_match on the combined workload (one rocprofv3 pass
# per counter group; the command and the per-step values are in the profiles
# folder).  Valid only for the kernel source they were measured on.
MATCH_COUNTERS = {
    "cfg5": {"source": "paper_2602_16100_amd/csrc/trace.hip",
             "sha256": "c9b11ae36f815781b39e2ccddb1fca6cd58dc757cfef139cb8fdfc38042cac7d",
             "SQ_INSTS_VALU_per_step": 3.895e8, "SQ_INSTS_SALU_per_step": 3.235e8},
}


# Issue counters of the instruction-bound kernels of two passes on the
# combined workload, per launch (one rocprofv3 pass; the command and values
# are in the profiles folder): the preferred-affinity evaluator of rows of at
# most three terms, and the path search.  Valid only for the kernel source
# they were measured on.
PASS_COUNTERS = {
    "k_pref_eval3": {"source": "paper_2602_16100_amd/csrc/select.hip",
                     "sha256": "3ba266f186a97c69f5525e79cbd1aa8e8de7774ba0177ee4f0f28a75ebc43f74",
                     "SQ_INSTS_VALU_per_launch": 1.1454e9, "SQ_INSTS_SALU_per_launch": 7.263e8},
    "k_ps_search": {"source": "paper_2602_16100_amd/csrc/paths.hip",
                    "sha256": "2cd6a2ef3bef6e4dbc6d79785967370e9c75b27ef64d4f64f685999d7c9ac81e",
                    "SQ_INSTS_VALU_per_launch": 4.129e9, "SQ_INSTS_SALU_per_launch": 3.355e9},
}


def issue_view(valu_instr, salu_instr, ms):
    """VALU issue (in lane-ops/s) against the chip's two wave-wide
    instructions per CU per clock, and the scalar unit's share of its one per
    CU per clock, from instruction counts over `ms` milliseconds."""
    lane_ops = valu_instr * 64 / (ms * 1e-3)
    return {"bound": "alu", "achieved": lane_ops, "peak": VALU_PEAK_LANE_OPS, "unit": "lane-ops/s",
            "frac": lane_ops / VALU_PEAK_LANE_OPS, "half_rate_peak": VALU_PEAK_LANE_OPS / 2,
            "salu_frac": salu_instr / (ms * 1e-3) / SALU_PEAK_INSTR,
            "source": "issue counters (profiles folder)"}


def alu_view(kernel, ms):
    """The issue-rate view of a kernel whose counters are recorded for its
    current source."""
    c = PASS_COUNTERS.get(kernel)
    if c is None or not source_unchanged(c) or not ms or ms <= 0:
        return None
    return {"kernel": kernel, **issue_view(c["SQ_INSTS_VALU_per_launch"], c["SQ_INSTS_SALU_per_launch"], ms)}


def source_unchanged(rec):
    import hashlib
    path = os.path.join(ROOT, rec["source"])
    if not os.path.exists(path):
        return False
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest() == rec["sha256"]


def measured_traffic(workload, kernel):
    """HBM bytes per launch from the FETCH_SIZE / WRITE_SIZE counter runs
    (scaled by a plain copy's readings), or None when the kernel's source
    has changed since they were taken."""
    import hashlib
    for t in TRAFFIC:
        if kernel not in t["bytes_per_launch"] or workload != t["workload"]:
            continue
        path = os.path.join(ROOT, t["source"])
        if not os.path.exists(path):
            return None
        with open(path, "rb") as f:
            if hashlib.sha256(f.read()).hexdigest() != t["sha256"]:
                return None
        return t["bytes_per_launch"][kernel]
    return None


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="cfg5", choices=["cfg5", "small", "cfg2", "cfg3", "cfg4"],
                    help="cfg5 (default): the combined step; cfg2 / cfg3 / cfg4: one stage on its own "
                         "configuration (selectors / flow tracing / masked reachability), one JSON line each")
    ap.add_argument("--variant", default="rpath", choices=["rpath", "prefix"],
                    help="cfg3 rule tables: compiled per-flow rules with i.i.d. care bits (rpath) or "
                         "destination-prefix routing tables with ports wildcarded (prefix)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target oracle time of the CPU baseline's sample (10-30 s keeps the run within minutes)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--only", default="all", choices=["all", "sel", "trace", "reach", "paths", "affinity", "preferred",
                                                     "synthesis", "update", "verdict", "delta"],
                    help="profiling aid: time one stage only (the JSON line then covers that stage); 'paths' "
                         "times only the pass with waypoint / forbidden-switch constraints, 'affinity' only the "
                         "node-affinity pass, 'preferred' only the preferred-affinity pass, 'synthesis' only the "
                         "path-synthesis pass, 'update' only the incremental re-evaluation, 'verdict' only the "
                         "verdict-only pass, 'delta' only the re-trace after rule changes")
    ap.add_argument("--no-paths", action="store_true",
                    help="skip the second timed pass with waypoint / forbidden-switch constraints")
    ap.add_argument("--no-affinity", action="store_true",
                    help="skip the timed pass of full node affinity over the same cluster")
    ap.add_argument("--no-rule-delta", action="store_true",
                    help="skip the timed incremental re-trace after rule changes")
    ap.add_argument("--no-preferred", action="store_true",
                    help="skip the timed pass of preferred node affinity (best feasible node per row)")
    ap.add_argument("--no-verdict-only", action="store_true",
                    help="skip the timed verdict-only pass (popcounts and endpoint probes instead of the bitset)")
    ap.add_argument("--no-update", action="store_true",
                    help="skip the timed incremental re-evaluation after node-label changes")
    ap.add_argument("--no-synthesis", action="store_true",
                    help="skip the timed pass of path synthesis over the same topology")
    ap.add_argument("--synthesis-requests", type=int, default=65536,
                    help="requests of the path-synthesis pass (the first flows of the workload)")
    ap.add_argument("--measure-valu", action="store_true",
                    help="measure the VALU and SALU issue rates, per instruction form, that the "
                         "instruction-issue rooflines are priced against")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="profiling aid: run a plain device copy of MIB MiB three times (HBM counter calibration)")
    ap.add_argument("--measure-plain", type=int, default=0, metavar="MIB",
                    help="profiling aid: time a plain device fill and a plain copy of MIB MiB (the rates an "
                         "HBM-bound kernel of that size can reach)")
    return ap.parse_args()


def measure_plain(mib, reps=10):
    """Torch's own fill and copy of MIB MiB, timed with events over `reps`
    launches after 2 untimed ones: the write-only and read+write rates a
    kernel that streams that many bytes can reach on this GPU."""
    import torch
    n = (mib << 20) // 8
    x = torch.empty(n, dtype=torch.int64, device="cuda:0")
    y = torch.ones(n, dtype=torch.int64, device="cuda:0")
    torch.cuda.synchronize()

    def timed(fn):
        for _ in range(2):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    fill_ms = timed(lambda: x.fill_(7))
    copy_ms = timed(lambda: x.copy_(y))
    b = n * 8
    print(json.dumps({"bytes": b, "fill_ms": fill_ms, "fill_gbs": b / fill_ms / 1e6,
                      "copy_ms": copy_ms, "copy_gbs": 2 * b / copy_ms / 1e6}), flush=True)


def measure_valu():
    """The chip's achieved wave-wide VALU (and one SALU) issue rate per
    instruction form (pc_measure_valu), with the shader clock read under that
    load, against the two VALU instructions per CU per clock the
    instruction-issue rooflines use."""
    import torch
    import paper_2602_16100_amd as pc
    torch.cuda.set_device(0)
    ctx = pc.Context(0)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    peak = VALU_PEAK_LANE_OPS / 64
    out = {"cus": cus, "peak_wave_instr_per_s": peak, "forms": {}}
    forms = ("add_sub_u32", "xor_b32", "and_or_b32_vvv", "and_or_b32_vvs", "lshlrev_b64", "add_sub_u32_e64",
             "s_xor_b32", "mov_b64", "cmp_ne_u32_e64", "cndmask_b32_e64", "bfi_b32", "xor_b32_sgpr", "mov_b32",
             "xor_b32_inline", "xor_b32_literal")
    for op, name in enumerate(forms):
        runs = [ctx.measure_valu(op, 10) for _ in range(3)]
        best, clock = max(runs)
        out["forms"][name] = {"wave_instr_per_s": [r for r, _ in runs], "clock_hz": [c for _, c in runs],
                              "best": best, "frac_of_peak": best / (SALU_PEAK_INSTR if name.startswith("s_") else peak),
                              "per_cu_per_clock": best / (cus * clock) if clock > 0 else None}
    print(json.dumps(out), flush=True)


def calibrate_copy(mib):
    """A plain elementwise copy (read n bytes, write n bytes) of known size,
    the yardstick the FETCH_SIZE / WRITE_SIZE counters are scaled by."""
    import torch
    n = mib << 20
    src = torch.ones(n // 4, dtype=torch.int32, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        torch.add(src, 0, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"calibrate_copy_bytes_read": n, "calibrate_copy_bytes_written": n, "launches": 3}), flush=True)


def make_workload(name):
    import synth
    if name == "cfg5":
        return synth.cfg5(paths=True), ("combined cross-layer validation, seed 4: 50,000 nodes x 64 labels; fat-tree k=48 "
                              "(2,880 switches), 16,384 rules/switch, 12 jurisdictions; 1,048,576 intents "
                              "(1/3 compute, 1/3 network, 1/3 hybrid); TTL 32; R-path rule tables")
    return (synth.combined_workload(7, 5000, 64, 16, 8, 2048, 30000, paths=True),
            "small combined workload (smoke scale)")


def sample_subproblem(wl, stride):
    """Every `stride`-th intent with the selector rows, traces and reach
    queries it references, renumbered into a standalone workload."""
    it = wl["intents"]
    idx = np.arange(0, it.shape[0], stride)
    sub = it[idx].copy()
    ex = wl["expect"][idx].copy()
    has_sel = (sub["kind"] & 1) == 1
    rows = sub["sel_row"][has_sel].astype(np.int32)
    sub["sel_row"][has_sel] = np.arange(rows.shape[0], dtype=np.int32)
    has_net = (sub["kind"] & 2) == 2
    tb, te = sub["trace_begin"][has_net], sub["trace_end"][has_net]
    lens = te - tb
    tidx = np.concatenate([np.arange(b, e) for b, e in zip(tb, te)]) if lens.sum() else np.zeros(0, np.int64)
    nb = np.zeros(lens.shape[0] + 1, np.int64)
    nb[1:] = np.cumsum(lens)
    sub["trace_begin"][has_net] = nb[:-1]
    sub["trace_end"][has_net] = nb[1:]
    q = ex["reach_q"]
    qsel = q >= 0
    qidx = q[qsel].astype(np.int64)
    ex["reach_q"][qsel] = np.arange(qidx.shape[0], dtype=np.int32)
    return dict(intents=sub, expect=ex, rows=rows, traces=tidx.astype(np.int64), queries=qidx)


def cpu_baseline(wl, pairs_total, target_s, gpu=None):
    """The oracle on every k-th intent (with the rows, traces and queries it
    references) on all the job's cores, k chosen so the sample takes about
    target_s, scaled to the whole job; the same on one thread for a smaller
    sample.  With the GPU's outputs, the all-cores sample is compared with
    them element by element."""
    import oracle
    threads = len(os.sched_getaffinity(0))
    env_cap = os.environ.get("OMP_NUM_THREADS")
    if env_cap and env_cap.isdigit():
        threads = min(threads, int(env_cap))

    def run(stride, nthreads):
        sp = sample_subproblem(wl, stride)
        t0 = time.perf_counter()
        feas, pc_, _ = oracle.selectors(wl["labels"], wl["pred_off"], wl["preds"], rows=sp["rows"],
                                        nthreads=nthreads)
        tr, _ = oracle.trace(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"], wl["rules"],
                             wl["hdr"], wl["ingress"], wl["ttl"], idx=sp["traces"], nthreads=nthreads)
        rc, _ = oracle.reach(wl["V"], wl["adj_off"], wl["adj"], wl["region"], wl["src"], wl["allowed"],
                             wl["target"], qidx=sp["queries"], nthreads=nthreads)
        _, reason, _, _ = oracle.report(sp["intents"], feas, pc_, wl["N"], tr, sp["expect"], rc)
        return time.perf_counter() - t0, sp, dict(feasible=feas, popcnt=pc_, traces=tr, reach=rc, reason=reason)

    def calibrated(nthreads, target):
        stride = 4096
        t, sp, res = run(stride, nthreads)
        # shrink the stride (at most 64x per probe) until the sample takes about target
        while t < target / 2 and stride > 1:
            stride = max(1, stride // 64, int(stride * max(t, 1e-3) / target))
            t, sp, res = run(stride, nthreads)
        return stride, t, sp, res

    I = wl["intents"].shape[0]
    stride, t, sp, res = calibrated(threads, target_s)
    frac = sp["intents"].shape[0] / I
    est_full = t / frac
    s1, t1, sp1, _ = calibrated(1, target_s / 2)
    est1 = t1 / (sp1["intents"].shape[0] / I)
    out = {
        "value": pairs_total / est_full,
        "unit": "selector evals/s (whole-job estimate)",
        "cores": threads,
        "kind": "oracle",
        "cpu_model": cpu_model(),
        "sample": (f"every {stride}th intent ({sp['intents'].shape[0]} of {I}: {sp['rows'].shape[0]} selector rows "
                   f"x {wl['N']} nodes, {sp['traces'].shape[0]} traces, {sp['queries'].shape[0]} reach queries, "
                   f"report) in {t:.2f} s on {threads} threads; whole job estimated at {est_full:.1f} s"),
        "est_step_s": est_full,
        "one_thread": {"value": pairs_total / est1, "cores": 1, "est_step_s": est1,
                       "sample": f"every {s1}th intent ({sp1['intents'].shape[0]} of {I}) in {t1:.2f} s"},
    }
    if gpu is not None:
        idx = np.arange(0, I, stride)
        checks = [("feasible", res["feasible"], gpu["feasible"][sp["rows"]]),
                  ("popcnt", res["popcnt"], gpu["popcnt"][sp["rows"]]),
                  ("reach", res["reach"], gpu["reach"][sp["queries"]]),
                  ("reason", res["reason"], gpu["reason"][idx])]
        for f in ("jmask", "last_switch", "last_port", "hops", "state"):
            checks.append((f"traces.{f}", res["traces"][f], gpu["traces"][f][sp["traces"]]))
        verdict = "bit-exact"
        for name, a, b in checks:
            if a.shape != b.shape or not np.array_equal(a, b):
                bad = np.argwhere(a != b) if a.shape == b.shape else None
                verdict = (f"MISMATCH in {name}" + (f" at {tuple(bad[0])}: oracle {a[tuple(bad[0])]} gpu "
                                                   f"{b[tuple(bad[0])]}" if bad is not None and bad.size else
                                                   f": shapes {a.shape} vs {b.shape}"))
                break
        out["parity"] = verdict
        out["parity_scope"] = (f"the all-cores sample ({sp['intents'].shape[0]} of {I} intents, "
                               f"{sp['rows'].shape[0]} selector rows, {sp['traces'].shape[0]} traces, "
                               f"{sp['queries'].shape[0]} reach queries) against the GPU's outputs of the last step")
    return out


HOP_KERNELS = ("k_tr_init", "k_tr_plan", "k_tr_scatter", "k_tr_match", "k_tr_walk")  # A3 after preparation


WALK_MAX = 8192  # the library's default switch-over to per-trace walks (PC_TRACE_WALK_MAX)


def trace_levels(wl, pc, ctx, D, full):
    """The hop levels the bucketed match kernel runs, with the switches each
    touches, from the library's own walk records (the first 8 switches of
    every walk; for later levels, a run with TTL l stops every trace that is
    still going at its level-l switch).  The library buckets level 0 when more than WALK_MAX traces
    start, and level l >= 1 when more than WALK_MAX traces entered level
    l - 1; later levels are walked per trace.  Returns the per-level
    (lookups, touched switches, rules of those switches) of the bucketed
    levels and the lookups of the walked ones."""
    import torch
    ing = wl["ingress"]
    S, T = wl["S"], wl["T"]
    started = (ing >= 0) & (ing < S)
    hops = full["hops"].astype(np.int64)
    R = np.diff(np.asarray(wl["rule_off"], np.int64))
    live = [int((started & (hops >= lv)).sum()) for lv in range(int(hops[started].max()) + 1)] if started.any() \
        else []
    bucketed = []
    for lv in range(len(live)):
        if (live[0] if lv == 0 else live[lv - 1]) > WALK_MAX:
            bucketed.append(lv)
        else:
            break
    out = torch.empty((T, 12), dtype=torch.uint8, device="cuda:0")
    vs = torch.empty(T, dtype=torch.int64, device="cuda:0")
    wk = torch.empty((T, 8), dtype=torch.int32, device="cuda:0")
    pc.pc_trace_flows_delta(S, D["port_off"], D["port_peer"], D["jur"], D["rule_off"], D["rules"], D["hdr"],
                            D["ingress"], wl["ttl"], out, vs, walk=wk, ctx=ctx)
    walk = wk.cpu().numpy()
    levels = []
    for lv in bucketed:
        if lv < 8:
            sw = walk[started & (hops >= lv), lv]
        else:  # past the walk records: a run with TTL lv stops every trace still going at its level-lv switch
            pc.pc_trace_flows(S, D["port_off"], D["port_peer"], D["jur"], D["rule_off"], D["rules"], D["hdr"],
                              D["ingress"], lv, out=out, ctx=ctx)
            sw = pc.records(out, pc.TRACE_OUT_DT)["last_switch"][started & (hops >= lv)]
        u = np.unique(sw)
        levels.append((live[lv], int(u.shape[0]), int(R[u].sum())))
    walked = int(sum(live[len(bucketed):]))
    return {"levels": levels, "walked_lookups": walked, "lookups": int(sum(live))}


def trace_roofline(wl, pc, ctx, D, full, prof, steps, workload):
    """k_tr_match, the hop loop's dominant kernel, against the HBM roofline
    with its algorithmic bytes: 30 B per rule of every switch a
    bucketed level touches, plus 32 B per trace (header, ingress, record).
    `layout_bytes` is what this library's layout needs for the same levels
    (384 B of chunk sets per 32-rule group).  The issue counters of the
    kernel, when recorded for its current source, give the ALU view."""
    lv = trace_levels(wl, pc, ctx, D, full)
    T = wl["T"]
    R = np.diff(np.asarray(wl["rule_off"], np.int64))
    rules = sum(r for _, _, r in lv["levels"])
    alg = rules * 30 + T * 32
    n, ms_tot = prof.get("k_tr_match", (0, 0.0))
    ms = ms_tot / steps
    gbs = alg / (ms * 1e-3) / 1e9 if ms > 0 else 0.0
    hop_ms = {k: prof[k][1] / steps for k in HOP_KERNELS if k in prof}
    out = {"kernel": "k_tr_match", "bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
           "frac": gbs / HBM_PEAK_GBS, "traffic": measured_traffic(workload, "k_tr_match"),
           "alg_bytes_per_step": alg, "launches_per_step": n / steps, "ms_per_step": ms,
           "bucketed_levels": [{"lookups": a, "switches": b, "rules": c} for a, b, c in lv["levels"]],
           "walked_lookups": lv["walked_lookups"],
           "hop_loop_ms_per_kernel": hop_ms, "hop_loop_ms": sum(hop_ms.values()),
           "hop_loop_frac": (alg / (sum(hop_ms.values()) * 1e-3) / 1e9 / HBM_PEAK_GBS) if hop_ms else None}
    c = MATCH_COUNTERS.get(workload)
    if c is not None and source_unchanged(c) and ms > 0:
        out["alu"] = issue_view(c["SQ_INSTS_VALU_per_step"], c["SQ_INSTS_SALU_per_step"], ms)
    return out


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def time_paths(args, wl, D, pc, ctx, feasible, popcnt):
    """Second timed pass: the same traces and queries with a required
    waypoint and two forbidden switches per flow (trace with watch lists,
    reachability through the waypoint avoiding the forbidden switches,
    verdict with the path checks).  The selector bitsets of the main pass
    are reused: the constraints do not touch them."""
    import torch
    dev = feasible.device
    T, Q, I = wl["T"], wl["Q"], wl["I"]
    traces = torch.empty((T, 12), dtype=torch.uint8, device=dev)
    visit = torch.empty(T, dtype=torch.int32, device=dev)
    reach = torch.empty(Q, dtype=torch.int32, device=dev)
    pass_ = torch.empty((I + 63) // 64, dtype=torch.int64, device=dev)
    reason = torch.empty(I, dtype=torch.uint8, device=dev)
    summary = torch.empty(pc.SUMMARY_BYTES, dtype=torch.uint8, device=dev)

    def step():
        pc.pc_trace_flows_watch(wl["S"], D["port_off"], D["port_peer"], D["jur"], D["rule_off"], D["rules"], D["hdr"],
                                D["ingress"], wl["ttl"], D["watch"], out=traces, visit=visit, ctx=ctx)
        pc.pc_masked_reach_via(wl["V"], D["adj_off"], D["adj"], D["region"], D["src"], D["allowed"], D["target"],
                               D["via"], D["forbid"], dist=reach, ctx=ctx)
        pc.pc_report_paths(D["intents"], feasible, popcnt, wl["N"], traces, D["expect"], reach, visit, D["pexp"],
                           pass_=pass_, reason=reason, summary=summary, ctx=ctx)

    elapsed, prof = timed_steps(args, ctx, step)

    def ktime(prefix):
        return sum(ms for name, (n, ms) in prof.items() if name.startswith(prefix)) / args.steps

    tr = pc.records(traces, pc.TRACE_OUT_DT)
    ing = wl["ingress"]
    started = (ing >= 0) & (ing < wl["S"])
    lookups = int((tr["hops"][started].astype(np.int64) + 1).sum())
    via = wl["via"]
    legs = int(Q + (via >= 0).sum())
    r = reason.cpu().numpy() & 0x7F
    out = {
        "constraints": "per flow: 1 required waypoint (on the compiled path with p=1/2), 2 forbidden switches "
                       "(each on the path with p=1/8); watch lists of 3 switches per trace",
        "ms_per_step": 1e3 * elapsed / args.steps,
        "entry_ms_per_step": {"pc_trace_flows_watch": ktime("k_tr_"), "pc_masked_reach_via": ktime("k_rc_"),
                              "pc_report_paths": ktime("k_report")},
        "flow_hops_per_s_kernel": lookups / (ktime("k_tr_") * 1e-3) if ktime("k_tr_") else None,
        "reach_legs_per_step": legs,
        "reach_legs_per_s_kernel": legs / (ktime("k_rc_") * 1e-3) if ktime("k_rc_") else None,
        "per_kernel": {name: {"launches_per_step": n / args.steps, "ms_per_step": ms / args.steps}
                       for name, (n, ms) in sorted(prof.items(), key=lambda kv: -kv[1][1])},
        "verdict": {"passed": int((r == 0).sum()), "forbidden_switch": int((r == 8).sum()),
                    "waypoint_missed": int((r == 9).sum()), "intents": I},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_paths(wl, 1e3 * elapsed / args.steps, args.cpu_seconds / 3)
    return out


def time_affinity(args, wl, pc, ctx, feasible):
    """Timed pass of full node affinity (pc_eval_affinity) over the same
    cluster: one required-affinity row per selector row (1-3 OR-ed terms of
    1-4 expressions, six operators), written into the same bitset shape."""
    import torch
    import synth
    dev = feasible.device
    I = feasible.shape[0]
    row_off, term_off, preds = synth.affinity_rows(wl.seed, wl.meta["cards"], I)
    D = {k: pc.to_device(v, dev) for k, v in (("labels", wl["labels"]), ("row_off", row_off),
                                               ("term_off", term_off), ("preds", preds))}
    popcnt = torch.empty(I, dtype=torch.int32, device=dev)
    unknown = torch.empty(I, dtype=torch.uint8, device=dev)

    def step():
        pc.pc_eval_affinity(D["labels"], D["row_off"], D["term_off"], D["preds"], feasible=feasible, popcnt=popcnt,
                            unknown=unknown, ctx=ctx)

    elapsed, prof = timed_steps(args, ctx, step)
    flags = ctx.data_errors(clear=True)
    N, L = wl["N"], wl["L"]
    W = (N + 63) // 64
    n_eval, eval_ms = prof["k_aff_eval"]
    avg_ms = eval_ms / max(n_eval, 1)
    n_terms, n_preds = term_off.shape[0] - 1, preds.shape[0]
    # the bitset, popcounts and inventory flags written; labels, expressions
    # and both offset arrays read once
    alg = I * W * 8 + I * 4 + I + n_preds * 40 + (n_terms + 1) * 4 + (I + 1) * 4 + N * L
    achieved = alg / (avg_ms * 1e-3) / 1e9
    pairs = I * N
    pcnt = popcnt.cpu().numpy()
    out = {
        "rows": I, "terms": int(n_terms), "expressions": int(n_preds),
        "ms_per_step": 1e3 * elapsed / args.steps,
        "evals_per_s": pairs * args.steps / elapsed,
        "per_kernel": {name: {"launches_per_step": n / args.steps, "ms_per_step": ms / args.steps}
                       for name, (n, ms) in sorted(prof.items(), key=lambda kv: -kv[1][1])},
        "roofline": {"kernel": "k_aff_eval", "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": measured_traffic(args.workload, "k_aff_eval"), "alg_bytes_per_launch": alg,
                     "avg_launch_ms": avg_ms},
        "feasible_rows": int((pcnt > 0).sum()),
        "unknown_rows": int((unknown.cpu().numpy() != 0).sum()),
        "data_error_flags": flags,
    }
    if not args.no_cpu_baseline:
        import oracle
        threads = len(os.sched_getaffinity(0))
        env_cap = os.environ.get("OMP_NUM_THREADS")
        if env_cap and env_cap.isdigit():
            threads = min(threads, int(env_cap))
        stride, t = 4096, 0.0
        while True:
            rows = np.arange(0, I, stride, dtype=np.int32)
            t0 = time.perf_counter()
            oracle.affinity(wl["labels"], row_off, term_off, preds, rows=rows, nthreads=threads)
            t = time.perf_counter() - t0
            if t >= args.cpu_seconds / 6 or stride == 1:
                break
            stride = max(1, stride // 64, int(stride * max(t, 1e-3) / (args.cpu_seconds / 3)))
        est = t * I / rows.shape[0]
        out["cpu_baseline"] = {"value": pairs / est, "unit": "affinity evals/s (whole-pass estimate)",
                               "cores": threads, "kind": "oracle",
                               "sample": f"every {stride}th row ({rows.shape[0]} of {I} rows x {N} nodes) in "
                                         f"{t:.2f} s; whole pass estimated at {est:.1f} s"}
    return out


def time_preferred(args, wl, pc, ctx, feasible):
    """Timed pass of preferred node affinity (pc_score_preferred) over the
    same cluster: per selector row 1-3 weighted terms (weights 1..100) of
    1-3 expressions, scored over the row's feasible nodes from the main
    pass's selector bitset."""
    import torch
    import synth
    dev = feasible.device
    I = feasible.shape[0]
    row_off, term_off, preds, weight = synth.preferred_rows(wl.seed, wl.meta["cards"], I)
    D = {k: pc.to_device(v, dev) for k, v in (("labels", wl["labels"]), ("row_off", row_off),
                                               ("term_off", term_off), ("preds", preds), ("weight", weight))}
    best = torch.empty(I, dtype=torch.int32, device=dev)
    score = torch.empty(I, dtype=torch.int32, device=dev)
    count = torch.empty(I, dtype=torch.int32, device=dev)

    def step():
        pc.pc_score_preferred(D["labels"], D["row_off"], D["term_off"], D["weight"], D["preds"], feasible=feasible,
                              best=best, score=score, count=count, ctx=ctx)

    elapsed, prof = timed_steps(args, ctx, step)
    flags = ctx.data_errors(clear=True)
    N, L = wl["N"], wl["L"]
    W = (N + 63) // 64
    # one evaluator launch per row class (8-bit scores, 16-bit scores,
    # decoded, at most three terms); together they read every row once, so
    # the roofline takes their summed time per step
    classes = ("k_pref_eval", "k_pref_eval16", "k_pref_decode", "k_pref_eval3")
    avg_ms = sum(prof[k][1] for k in classes if k in prof) / args.steps
    n_terms, n_preds = term_off.shape[0] - 1, preds.shape[0]
    # the feasible bitset, expressions, weights, offsets and labels read
    # once; best node, score and tie count written
    alg = I * W * 8 + I * 12 + n_preds * 40 + n_terms * 4 + (n_terms + 1) * 4 + (I + 1) * 4 + N * L
    achieved = alg / (avg_ms * 1e-3) / 1e9
    pairs = I * N
    b = best.cpu().numpy()
    out = {
        "rows": I, "terms": int(n_terms), "expressions": int(n_preds),
        "ms_per_step": 1e3 * elapsed / args.steps,
        "evals_per_s": pairs * args.steps / elapsed,
        "per_kernel": {name: {"launches_per_step": n / args.steps, "ms_per_step": ms / args.steps}
                       for name, (n, ms) in sorted(prof.items(), key=lambda kv: -kv[1][1])},
        "roofline": {"kernel": "+".join(classes), "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": measured_traffic(args.workload, "k_pref_eval"), "alg_bytes_per_launch": alg,
                     "avg_launch_ms": avg_ms,
                     # the class that takes every row at this size is instruction bound
                     "alu": alu_view("k_pref_eval3", prof["k_pref_eval3"][1] / max(prof["k_pref_eval3"][0], 1)
                                     if "k_pref_eval3" in prof else None)},
        "placed_rows": int((b >= 0).sum()),
        "mean_best_score": float(score.cpu().numpy()[b >= 0].mean()) if (b >= 0).any() else 0.0,
        "data_error_flags": flags,
    }
    if not args.no_cpu_baseline:
        import oracle
        threads = len(os.sched_getaffinity(0))
        env_cap = os.environ.get("OMP_NUM_THREADS")
        if env_cap and env_cap.isdigit():
            threads = min(threads, int(env_cap))
        fh = feasible.cpu().numpy().view(np.uint64)
        stride, t = 4096, 0.0
        while True:
            rows = np.arange(0, I, stride, dtype=np.int32)
            t0 = time.perf_counter()
            oracle.preferred(wl["labels"], row_off, term_off, weight, preds, feasible=fh, rows=rows, nthreads=threads)
            t = time.perf_counter() - t0
            if t >= args.cpu_seconds / 6 or stride == 1:
                break
            stride = max(1, stride // 64, int(stride * max(t, 1e-3) / (args.cpu_seconds / 3)))
        est = t * I / rows.shape[0]
        out["cpu_baseline"] = {"value": pairs / est, "unit": "preferred-affinity evals/s (whole-pass estimate)",
                               "cores": threads, "kind": "oracle",
                               "sample": f"every {stride}th row ({rows.shape[0]} of {I} rows x {N} nodes) in "
                                         f"{t:.2f} s; whole pass estimated at {est:.1f} s"}
    return out


def time_verdict_only(args, wl, pc, ctx, D, traces, reach):
    """Verdict-only pass: the selector rows' popcounts without the bitset
    (pc_eval_selectors_count), the hybrid intents' endpoint bits as probes
    (pc_probe_selectors) and the verdict from both (pc_report_counts), on the
    traces and reach distances of the main pass.  Its verdict must equal the
    main pass's."""
    import torch
    dev = traces.device
    it = wl["intents"]
    I = it.shape[0]
    hyb = it["kind"] == 3
    sel = np.repeat(hyb, 2)
    rows = np.repeat(it["sel_row"], 2)[sel].astype(np.int32)
    nodes = np.stack([it["src_node"], it["dst_node"]], axis=1).reshape(-1)[sel].astype(np.int32)
    pos = pc.to_device(np.flatnonzero(sel).astype(np.int64), dev)
    Dr, Dn = pc.to_device(rows, dev), pc.to_device(nodes, dev)
    popcnt = torch.empty(wl["I_rows"], dtype=torch.int32, device=dev)
    bits = torch.empty(rows.shape[0], dtype=torch.uint8, device=dev)
    ends = torch.zeros(2 * I, dtype=torch.uint8, device=dev)
    pass_ = torch.empty((I + 63) // 64, dtype=torch.int64, device=dev)
    reason = torch.empty(I, dtype=torch.uint8, device=dev)
    summary = torch.empty(pc.SUMMARY_BYTES, dtype=torch.uint8, device=dev)

    def step():
        pc.pc_eval_selectors_count(D["labels"], D["pred_off"], D["preds"], popcnt=popcnt, ctx=ctx)
        pc.pc_probe_selectors(D["labels"], D["pred_off"], D["preds"], Dr, Dn, bits=bits, ctx=ctx)
        ends.index_copy_(0, pos, bits)
        pc.pc_report_counts(D["intents"], popcnt, wl["N"], ends, traces, D["expect"], reach, pass_=pass_,
                            reason=reason, summary=summary, ctx=ctx)

    elapsed, prof = timed_steps(args, ctx, step)
    return {"ms_per_step": 1e3 * elapsed / args.steps,
            "per_kernel": {name: {"launches_per_step": n / args.steps, "ms_per_step": ms / args.steps}
                           for name, (n, ms) in sorted(prof.items(), key=lambda kv: -kv[1][1])},
            "probes": int(rows.shape[0]),
            "_pass": pass_, "_reason": reason}


def time_update(args, wl, pc, ctx, D, feasible, popcnt):
    """Incremental re-evaluation (pc_update_nodes) after relabelling M random
    nodes of the cluster, against the full pc_eval_selectors of the new
    labels.  The bitsets are brought to the old labels' state before each
    timed call; the timed region is the call alone.  Above W / 32 nodes the
    library itself takes the full evaluation."""
    import torch
    dev = feasible.device
    rng = np.random.default_rng([wl.seed, 15])
    N, L, I = wl["N"], wl["L"], feasible.shape[0]
    W = (N + 63) // 64
    cards = wl.meta["cards"]
    labels = wl["labels"]
    base = pc.to_device(labels, dev)
    out = {"rows": I, "nodes": N, "full_above": W // 32, "per_m": {}}
    for M in (1, 16, 64, 1024):
        nodes = rng.choice(N, size=M, replace=False).astype(np.int32)
        new = labels.copy()
        new[nodes] = rng.integers(0, cards[None, :], size=(M, L)).astype(np.uint8)
        Dn = pc.to_device(new, dev)
        Dnodes = pc.to_device(nodes, dev)
        t_upd, t_full = [], []
        for it in range(args.warmup + args.steps):
            pc.pc_eval_selectors(base, D["pred_off"], D["preds"], feasible=feasible, popcnt=popcnt, ctx=ctx)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            pc.pc_update_nodes(Dn, D["pred_off"], D["preds"], Dnodes, feasible, popcnt, ctx=ctx)
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            pc.pc_eval_selectors(Dn, D["pred_off"], D["preds"], feasible=feasible, popcnt=popcnt, ctx=ctx)
            torch.cuda.synchronize()
            t2 = time.perf_counter()
            if it >= args.warmup:
                t_upd.append(t1 - t0)
                t_full.append(t2 - t1)
        u, f = float(np.median(t_upd)), float(np.median(t_full))
        out["per_m"][str(M)] = {"ms_per_update": 1e3 * u, "ms_full_evaluation": 1e3 * f, "speedup": f / u,
                                "path": "incremental" if M <= W // 32 else "full re-evaluation"}
    if not args.no_cpu_baseline:
        import oracle
        threads = len(os.sched_getaffinity(0))
        env_cap = os.environ.get("OMP_NUM_THREADS")
        if env_cap and env_cap.isdigit():
            threads = min(threads, int(env_cap))
        nodes = rng.choice(N, size=64, replace=False).astype(np.int32)
        R = min(I, 65536)  # the first R rows: the oracle's copies of the bitset stay small
        f0 = feasible[:R].cpu().numpy().view(np.uint64)
        p0 = popcnt[:R].cpu().numpy().view(np.uint32)
        t0 = time.perf_counter()
        oracle.update_nodes(labels, wl["pred_off"][:R + 1], wl["preds"], nodes, f0, p0, nthreads=threads)
        t = (time.perf_counter() - t0) * I / R
        out["cpu_baseline"] = {"value": 1.0 / t, "unit": "updates/s (64 relabelled nodes, all rows; estimate)",
                               "cores": threads, "kind": "oracle",
                               "sample": f"one update of 64 nodes over the first {R} of {I} rows, scaled to all rows: "
                                         f"{t:.3f} s per update"}
    return out


def time_rule_delta(args, wl, pc, ctx, D):
    """Incremental re-trace (pc_trace_flows_delta, with walk records) after
    rewriting the rules of 1 core switch, 1 edge switch and 16 random
    switches of the combined workload's fat-tree, against a full
    pc_trace_flows on the new tables.  The previous records, summaries and
    walk records are restored before each timed call; the timed region is
    the call alone.  The context declares the keep-tables promise (tables
    change only in the listed switches between calls), so each delta
    re-prepares only its listed switches; each change starts from a context
    whose kept prepared tables are the original ones."""
    import torch
    import synth
    ctx.keep_tables(True)
    dev = D["ingress"].device
    S, T, ttl = wl["S"], wl["T"], wl["ttl"]
    out0 = torch.empty((T, 12), dtype=torch.uint8, device=dev)
    vs0 = torch.empty(T, dtype=torch.int64, device=dev)
    wk0 = torch.empty((T, 8), dtype=torch.int32, device=dev)
    pc.pc_trace_flows_delta(S, D["port_off"], D["port_peer"], D["jur"], D["rule_off"], D["rules"], D["hdr"],
                            D["ingress"], ttl, out0, vs0, walk=wk0, ctx=ctx)
    out, vs, wk = out0.clone(), vs0.clone(), wk0.clone()
    k = int(round((4 * S / 5) ** 0.5))  # fat-tree: S = 5 k^2 / 4
    rng = np.random.default_rng([wl.seed, 17])
    cases = {"1 core switch": np.array([k * k + 7], np.int32), "1 edge switch": np.array([3 * k + 1], np.int32),
             "16 switches": rng.choice(S, size=16, replace=False).astype(np.int32)}
    res = {"traces": T, "switches": S, "per_change": {}}
    vs_host = vs0.cpu().numpy().view(np.uint64)
    wk_host = wk0.cpu().numpy()
    short_host = pc.records(out0, pc.TRACE_OUT_DT)["hops"].astype(np.int64) + 1 <= 8
    for name, changed in cases.items():
        r_off, rules = synth.mutate_tables(wl.seed, wl["port_off"], wl["rule_off"], wl["rules"], changed)
        Dr = {"rule_off": pc.to_device(r_off, dev), "rules": pc.to_device(rules, dev)}
        Dc = pc.to_device(changed, dev)
        t_d, t_f = [], []
        n = None
        # the context's kept tables go back to the original ones: a delta call
        # may re-prepare only the switches it lists
        pc.pc_trace_flows_delta(S, D["port_off"], D["port_peer"], D["jur"], D["rule_off"], D["rules"], D["hdr"],
                                D["ingress"], ttl, out, vs, walk=wk, ctx=ctx)
        for it in range(args.warmup + args.steps):
            out.copy_(out0)
            vs.copy_(vs0)
            wk.copy_(wk0)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            n = pc.pc_trace_flows_delta(S, D["port_off"], D["port_peer"], D["jur"], Dr["rule_off"], Dr["rules"],
                                        D["hdr"], D["ingress"], ttl, out, vs, changed=Dc, walk=wk, ctx=ctx)
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            pc.pc_trace_flows(S, D["port_off"], D["port_peer"], D["jur"], Dr["rule_off"], Dr["rules"], D["hdr"],
                              D["ingress"], ttl, ctx=ctx)
            torch.cuda.synchronize()
            t2 = time.perf_counter()
            if it >= args.warmup:
                t_d.append(t1 - t0)
                t_f.append(t2 - t1)
        d, f = float(np.median(t_d)), float(np.median(t_f))
        m = 0
        for sw in changed:
            m |= 1 << (int(sw) & 63)
        entry = {"retraced": int(n.cpu().numpy()[0]), "ms_per_delta": 1e3 * d, "ms_full_trace": 1e3 * f,
                 "speedup": f / d}
        if not args.no_cpu_baseline:
            import oracle
            threads = len(os.sched_getaffinity(0))
            env_cap = os.environ.get("OMP_NUM_THREADS")
            if env_cap and env_cap.isdigit():
                threads = min(threads, int(env_cap))
            sel = np.flatnonzero(np.where(short_host, np.isin(wk_host, changed).any(axis=1),
                                          (vs_host & np.uint64(m)) != 0))
            samp = sel[:: max(1, sel.shape[0] // 20000)]
            t0 = time.perf_counter()
            oracle.trace(S, wl["port_off"], wl["port_peer"], wl["jur"], r_off, rules, wl["hdr"], wl["ingress"], ttl,
                         idx=samp, nthreads=threads)
            t = (time.perf_counter() - t0) * sel.shape[0] / max(samp.shape[0], 1)
            entry["cpu_baseline"] = {"value": 1.0 / t if t > 0 else None,
                                     "unit": "deltas/s (the oracle re-tracing the selected traces; estimate)",
                                     "cores": threads, "kind": "oracle",
                                     "sample": f"{samp.shape[0]} of the {sel.shape[0]} selected traces, scaled: "
                                               f"{t:.3f} s per delta"}
        res["per_change"][name] = entry
    ctx.keep_tables(False)
    return res


def time_synthesis(args, wl, pc, ctx):
    """Timed pass of path synthesis (pc_synthesize_paths) over the same
    topology: the first flows' endpoints, allowed jurisdictions, waypoint,
    forbidden switches, keys and egress ports, with link weights 1..10
    (weighted search), at most `ttl` links per walk."""
    import torch
    import synth
    dev = "cuda:0"
    Q = min(args.synthesis_requests, wl["Q"])
    ex = wl["expect"]
    has = ex["reach_q"] >= 0
    out_port = np.zeros(wl["Q"], np.int32)
    out_port[ex["reach_q"][has]] = ex["dst_port"][has]
    weight = synth.port_weights(wl.seed, wl["port_peer"].shape[0])
    arr = dict(src=wl["src"][:Q], target=wl["target"][:Q], allowed=wl["allowed"][:Q], via=wl["via"][:Q],
               forbid=wl["forbid"][:Q], key=wl["hdr"][:Q], out_port=out_port[:Q])
    D = {k: pc.to_device(np.ascontiguousarray(v), dev) for k, v in arr.items()}
    T = {k: pc.to_device(wl[k], dev) for k in ("port_off", "port_peer", "jur")}
    Wd = pc.to_device(weight, dev)
    S, ttl, prio = wl["S"], wl["ttl"], 40000
    slots = ttl + 1
    hops = torch.empty(Q, dtype=torch.int32, device=dev)
    path = torch.empty((Q, slots), dtype=torch.int32, device=dev)
    rules = torch.empty((Q, slots, 40), dtype=torch.uint8, device=dev)

    def step():
        pc.pc_synthesize_paths(S, T["port_off"], T["port_peer"], T["jur"], D["src"], D["target"], D["allowed"],
                               D["via"], D["forbid"], D["key"], D["out_port"], prio, ttl, weight=Wd, hops=hops,
                               path=path, rules=rules, ctx=ctx)

    elapsed, prof = timed_steps(args, ctx, step)
    flags = ctx.data_errors(clear=True)
    h = hops.cpu().numpy()
    legs = int(Q + (arr["via"] >= 0).sum())
    out = {
        "requests": Q, "legs": legs, "weights": "uniform 1..10 per port", "max_hops": ttl,
        "ms_per_step": 1e3 * elapsed / args.steps,
        "paths_per_s": Q * args.steps / elapsed,
        "per_kernel": {name: {"launches_per_step": n / args.steps, "ms_per_step": ms / args.steps}
                       for name, (n, ms) in sorted(prof.items(), key=lambda kv: -kv[1][1])},
        "synthesized": int((h >= 0).sum()),
        "mean_hops": float(h[h >= 0].mean()) if (h >= 0).any() else None,
        "data_error_flags": flags,
        # the search is instruction and latency bound (no HBM stream to
        # price): its issue rate, when counters are recorded for its source
        "roofline": alu_view("k_ps_search", prof["k_ps_search"][1] / max(prof["k_ps_search"][0], 1)
                             if "k_ps_search" in prof else None),
    }
    if not args.no_cpu_baseline:
        import oracle
        threads = len(os.sched_getaffinity(0))
        env_cap = os.environ.get("OMP_NUM_THREADS")
        if env_cap and env_cap.isdigit():
            threads = min(threads, int(env_cap))
        stride = 1024
        while True:
            qidx = np.arange(0, Q, stride, dtype=np.int64)
            t0 = time.perf_counter()
            oracle.synthesize(S, wl["port_off"], wl["port_peer"], wl["jur"], arr["src"], arr["target"],
                              arr["allowed"], arr["via"], arr["forbid"], arr["key"], arr["out_port"], prio, ttl,
                              weight=weight, qidx=qidx, nthreads=threads)
            t = time.perf_counter() - t0
            if t >= args.cpu_seconds / 6 or stride == 1:
                break
            stride = max(1, stride // 64, int(stride * max(t, 1e-3) / (args.cpu_seconds / 3)))
        est = t * Q / qidx.shape[0]
        out["cpu_baseline"] = {"value": Q / est, "unit": "synthesized paths/s (whole-pass estimate)",
                               "cores": threads, "kind": "oracle",
                               "sample": f"every {stride}th request ({qidx.shape[0]} of {Q}) in {t:.2f} s; whole "
                                         f"pass estimated at {est:.1f} s"}
    return out


def cpu_baseline_paths(wl, gpu_ms, target_s):
    """The oracle on every k-th flow of the constrained pass (traces with
    watch lists and waypoint reach), scaled to the whole pass."""
    import oracle
    threads = len(os.sched_getaffinity(0))
    env_cap = os.environ.get("OMP_NUM_THREADS")
    if env_cap and env_cap.isdigit():
        threads = min(threads, int(env_cap))
    T = wl["T"]

    def run(stride):
        idx = np.arange(0, T, stride, dtype=np.int64)
        t0 = time.perf_counter()
        oracle.trace(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"], wl["rules"], wl["hdr"],
                     wl["ingress"], wl["ttl"], idx=idx, nthreads=threads, watch=wl["watch"])
        oracle.reach_via(wl["V"], wl["adj_off"], wl["adj"], wl["region"], wl["src"], wl["allowed"], wl["target"],
                         wl["via"], wl["forbid"], qidx=idx, nthreads=threads)
        return time.perf_counter() - t0, idx.shape[0]

    stride = 4096
    t, n = run(stride)
    while t < target_s / 2 and stride > 1:
        stride = max(1, stride // 64, int(stride * max(t, 1e-3) / target_s))
        t, n = run(stride)
    est = t * T / n
    return {"value": T / est, "unit": "constrained flows (trace + waypoint reach) per second, whole-pass estimate",
            "cores": threads, "kind": "oracle",
            "sample": f"every {stride}th flow ({n} of {T} traces and reach queries) in {t:.2f} s; whole pass "
                      f"estimated at {est:.1f} s against {gpu_ms:.2f} ms on the GPU"}


def oracle_threads():
    threads = len(os.sched_getaffinity(0))
    env_cap = os.environ.get("OMP_NUM_THREADS")
    if env_cap and env_cap.isdigit():
        threads = min(threads, int(env_cap))
    return threads


def timed_steps(args, ctx, step):
    """W warm-up steps, then K steps timed by the host clock with nothing
    but the step on the stream, then K more steps with the per-kernel
    profiler on (its event pair around every launch adds a gap of several
    microseconds per kernel, so those steps are not the ones timed);
    returns (seconds of the K plain steps, {kernel: (launches, ms)})."""
    import torch
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ctx.data_errors(clear=True)
    ctx.profile(False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ctx.profile(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    prof = ctx.profile_read()
    ctx.profile(False)
    return t1 - t0, prof


def single_line(args, desc, value, unit, elapsed, config, roofline, extra):
    line = {"metric": "flow hops traced/sec + selector evals/sec on 1 MI355X; % of peak HBM GB/s",
            "value": value, "unit": unit, "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
            "ms_per_step": 1e3 * elapsed / args.steps, "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "u64 bitsets / int32 (integer work, no floating point)",
            "data": "synthetic (seeded generators; no dataset)",
            "config": dict({"workload": desc, "parallelism": "single GPU"}, **config), "roofline": roofline}
    line.update(extra)
    return line


def per_kernel_table(prof, steps):
    return {name: {"launches_per_step": n / steps, "ms_per_step": ms / steps}
            for name, (n, ms) in sorted(prof.items(), key=lambda kv: -kv[1][1])}


def bench_cfg2(args, pc, ctx):
    """Selector evaluation on its own: 100,000 nodes x 64 labels, 16,384 rows."""
    import synth
    import torch
    wl = synth.cfg2()
    desc = ("selector evaluation, seed 1: 100,000 nodes x 64 labels (cardinality from {2,4,16,64}); 16,384 rows "
            "of 1-8 In / NotIn / Exists predicates")
    D = {k: pc.to_device(wl[k], "cuda:0") for k in ("labels", "pred_off", "preds")}
    N, L, I = wl["N"], wl["L"], wl["I_rows"]
    W = (N + 63) // 64
    feas = torch.empty((I, W), dtype=torch.int64, device="cuda:0")
    pop = torch.empty(I, dtype=torch.int32, device="cuda:0")
    step = lambda: pc.pc_eval_selectors(D["labels"], D["pred_off"], D["preds"], feasible=feas, popcnt=pop,  # noqa
                                        ctx=ctx)
    elapsed, prof = timed_steps(args, ctx, step)
    n, ms = prof["k_sel_eval"]
    avg = ms / n
    alg = I * W * 8 + I * 4 + wl["n_preds"] * 40 + N * L
    gbs = alg / (avg * 1e-3) / 1e9
    pairs = I * N
    extra = {"per_kernel": per_kernel_table(prof, args.steps),
             "kernel_rate_evals_per_s": pairs / (avg * 1e-3),
             "data_error_flags": ctx.data_errors(clear=True)}
    roof = {"kernel": "k_sel_eval", "bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": gbs / HBM_PEAK_GBS, "traffic": measured_traffic(args.workload, "k_sel_eval"), "alg_bytes_per_launch": alg, "avg_launch_ms": avg,
            "floor_us_at_peak": alg / (HBM_PEAK_GBS * 1e9) * 1e6}
    if not args.no_cpu_baseline:
        import oracle
        th = oracle_threads()
        stride = 16
        rows = np.arange(0, I, stride, dtype=np.int32)
        t0 = time.perf_counter()
        fo, po, _ = oracle.selectors(wl["labels"], wl["pred_off"], wl["preds"], rows=rows, nthreads=th)
        t = (time.perf_counter() - t0) * stride
        t1s0 = time.perf_counter()
        oracle.selectors(wl["labels"], wl["pred_off"], wl["preds"], rows=rows[::16], nthreads=1)
        t1 = (time.perf_counter() - t1s0) * stride * 16
        fg = feas.cpu().numpy().view(np.uint64)[rows]
        pg = pop.cpu().numpy().view(np.uint32)[rows]
        extra["cpu_baseline"] = {"value": pairs / t, "unit": "selector evals/s (whole-job estimate)", "cores": th,
                                 "kind": "oracle", "cpu_model": cpu_model(),
                                 "sample": f"every {stride}th row ({rows.shape[0]} of {I}) in {t / stride:.2f} s",
                                 "one_thread": {"value": pairs / t1, "cores": 1,
                                                "sample": f"every {stride * 16}th row"},
                                 "parity": "bit-exact" if np.array_equal(fg, fo) and np.array_equal(pg, po)
                                 else "MISMATCH", "parity_scope": "the sampled rows"}
    return single_line(args, desc, pairs * args.steps / elapsed, "selector evals/s ((row,node) pairs per second)",
                       elapsed, {"rows": I, "nodes": N, "labels": L}, roof, extra)


def bench_cfg3(args, pc, ctx):
    """Flow tracing on its own: fat-tree k=32, 4,096 rules per switch, 4.19 M traces."""
    import synth
    import torch
    wl = synth.cfg3(variant=args.variant)
    tables = ("per-flow compiled rules with 30% wildcard bits" if args.variant == "rpath" else
              "destination-prefix routing tables (16-32 bit prefixes; ports, source, protocol wildcarded)")
    desc = (f"flow tracing, seed 2: fat-tree k=32 (1,280 switches), 4,096 rules per switch ({tables}), "
            f"4,194,304 headers at edge switches, TTL 32")
    D = {k: pc.to_device(wl[k], "cuda:0") for k in ("port_off", "port_peer", "jur", "rule_off", "rules", "hdr",
                                                     "ingress")}
    T = wl["T"]
    out = torch.empty((T, 12), dtype=torch.uint8, device="cuda:0")
    step = lambda: pc.pc_trace_flows(wl["S"], D["port_off"], D["port_peer"], D["jur"], D["rule_off"],  # noqa
                                     D["rules"], D["hdr"], D["ingress"], wl["ttl"], out=out, ctx=ctx)
    elapsed, prof = timed_steps(args, ctx, step)
    tr = pc.records(out, pc.TRACE_OUT_DT)
    ing = wl["ingress"]
    started = (ing >= 0) & (ing < wl["S"])
    lookups = int((tr["hops"][started].astype(np.int64) + 1).sum())
    roof = trace_roofline(wl, pc, ctx, D, tr, prof, args.steps, f"cfg3-{args.variant}")
    prep_ms = sum(ms for k, (n, ms) in prof.items() if k in ("k_tr_prep", "k_tr_choose", "k_tr_switch_info",
                                                             "k_tr_port_check")) / args.steps
    extra = {"per_kernel": per_kernel_table(prof, args.steps), "flow_lookups_per_step": lookups,
             "mean_lookups_per_trace": lookups / max(int(started.sum()), 1),
             "terminal_states": {k: int((tr["state"] == v).sum()) for k, v in
                                 (("egress", 0), ("drop", 1), ("miss", 2), ("ttl", 3))},
             "hop_loop_lookups_per_s": lookups / (roof["hop_loop_ms"] * 1e-3) if roof["hop_loop_ms"] else None,
             "prep_ms_per_step": prep_ms, "data_error_flags": ctx.data_errors(clear=True)}
    if not args.no_cpu_baseline:
        import oracle
        th = oracle_threads()
        stride = 64
        idx = np.arange(0, T, stride)
        t0 = time.perf_counter()
        to, _ = oracle.trace(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"], wl["rules"],
                             wl["hdr"], wl["ingress"], wl["ttl"], idx=idx, nthreads=th)
        t = (time.perf_counter() - t0) * stride
        t1s0 = time.perf_counter()
        oracle.trace(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"], wl["rules"], wl["hdr"],
                     wl["ingress"], wl["ttl"], idx=idx[::16], nthreads=1)
        t1 = (time.perf_counter() - t1s0) * stride * 16
        same = all(np.array_equal(tr[f][idx], to[f]) for f in ("jmask", "last_switch", "last_port", "hops", "state"))
        extra["cpu_baseline"] = {"value": lookups / t, "unit": "flow lookups/s (whole-job estimate)", "cores": th,
                                 "kind": "oracle", "cpu_model": cpu_model(),
                                 "sample": f"every {stride}th trace ({idx.shape[0]} of {T}) in {t / stride:.2f} s",
                                 "one_thread": {"value": lookups / t1, "cores": 1,
                                                "sample": f"every {stride * 16}th trace"},
                                 "parity": "bit-exact" if same else "MISMATCH", "parity_scope": "the sampled traces"}
    return single_line(args, desc, lookups * args.steps / elapsed,
                       "flow lookups/s (hops + 1 per trace, per second of whole-call time incl. table preparation)",
                       elapsed, {"switches": wl["S"], "rules": wl["n_rules"], "traces": T, "ttl": wl["ttl"],
                                 "variant": args.variant}, roof, extra)


def bench_cfg4(args, pc, ctx):
    """Masked reachability on its own: 1,000,000-vertex RGG, 256 full-row queries."""
    import synth
    import torch
    wl = synth.cfg4()
    desc = ("masked reachability, seed 3: random geometric graph of 1,000,000 switches (mean degree 4), "
            "16-region Voronoi map, 256 queries of 1-8 allowed regions, full distance rows")
    D = {k: pc.to_device(wl[k], "cuda:0") for k in ("adj_off", "adj", "region", "src", "allowed")}
    V, Q = wl["V"], wl["Q"]
    dist = torch.empty((Q, V), dtype=torch.int32, device="cuda:0")
    step = lambda: pc.pc_masked_reach(V, D["adj_off"], D["adj"], D["region"], D["src"], D["allowed"],  # noqa
                                      dist=dist, ctx=ctx)
    elapsed, prof = timed_steps(args, ctx, step)
    per_k = per_kernel_table(prof, args.steps)
    fill = per_k.get("k_fill_u32", {}).get("ms_per_step")
    ms = sum(v["ms_per_step"] for v in per_k.values())
    store = Q * V * 4
    alg = store + (V + 1) * 4 + int(wl["adj"].shape[0]) * 4 + V
    gbs = alg / (ms * 1e-3) / 1e9
    roof = {"kernel": "+".join(per_k), "bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": gbs / HBM_PEAK_GBS, "traffic": measured_traffic("cfg4", "pc_masked_reach"),
            "alg_bytes_per_launch": alg, "avg_launch_ms": ms, "floor_us_at_peak": alg / (HBM_PEAK_GBS * 1e9) * 1e6}
    extra = {"per_kernel": per_k, "fill_ms": fill,
             "fill_gbs": store / (fill * 1e-3) / 1e9 if fill else None,
             "data_error_flags": ctx.data_errors(clear=True)}
    d = dist.cpu().numpy()
    extra["reached_per_query_mean"] = float((d >= 0).sum(1).mean())
    if not args.no_cpu_baseline:
        import oracle
        th = oracle_threads()
        t0 = time.perf_counter()
        do, _ = oracle.reach(V, wl["adj_off"], wl["adj"], wl["region"], wl["src"], wl["allowed"], nthreads=th)
        t = time.perf_counter() - t0
        t1s0 = time.perf_counter()
        qs = np.arange(0, Q, 16)
        oracle.reach(V, wl["adj_off"], wl["adj"], wl["region"], wl["src"], wl["allowed"], qidx=qs, nthreads=1)
        t1 = (time.perf_counter() - t1s0) * 16
        extra["cpu_baseline"] = {"value": Q * V / t, "unit": "(query, vertex) distances/s", "cores": th,
                                 "kind": "oracle", "cpu_model": cpu_model(),
                                 "sample": f"all {Q} queries in {t:.2f} s",
                                 "one_thread": {"value": Q * V / t1, "cores": 1, "sample": "every 16th query"},
                                 "parity": "bit-exact" if np.array_equal(d, do) else "MISMATCH",
                                 "parity_scope": "every distance row"}
    return single_line(args, desc, Q * V * args.steps / elapsed, "(query, vertex) distances/s", elapsed,
                       {"vertices": V, "queries": Q}, roof, extra)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (the check shards by intent, with no exchange between GPUs); "
              f"--gpus {args.gpus} is not supported", file=sys.stderr)
        sys.exit(2)

    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return
    if args.measure_plain:
        measure_plain(args.measure_plain)
        return
    if args.measure_valu:
        measure_valu()
        return

    import torch
    import paper_2602_16100_amd as pc

    if args.workload in ("cfg2", "cfg3", "cfg4"):
        torch.cuda.set_device(0)
        ctx = pc.context(0)
        fn = {"cfg2": bench_cfg2, "cfg3": bench_cfg3, "cfg4": bench_cfg4}[args.workload]
        print(json.dumps(fn(args, pc, ctx)), flush=True)
        return

    wl, desc = make_workload(args.workload)
    dev = "cuda:0"
    torch.cuda.set_device(0)
    D = {k: pc.to_device(v, dev) for k, v in wl.arrays.items() if isinstance(v, np.ndarray) and k != "pts"}
    N, L = wl["N"], wl["L"]
    I_rows = wl["I_rows"]
    W = (N + 63) // 64
    I = wl["I"]
    T = wl["T"]
    Q = wl["Q"]
    feasible = torch.empty((I_rows, W), dtype=torch.int64, device=dev)
    popcnt = torch.empty(I_rows, dtype=torch.int32, device=dev)
    traces = torch.empty((T, 12), dtype=torch.uint8, device=dev)
    reach = torch.empty(Q, dtype=torch.int32, device=dev)
    pass_ = torch.empty((I + 63) // 64, dtype=torch.int64, device=dev)
    reason = torch.empty(I, dtype=torch.uint8, device=dev)
    summary = torch.empty(pc.SUMMARY_BYTES, dtype=torch.uint8, device=dev)
    ctx = pc.context(0)

    only = args.only
    if only == "affinity":
        print(json.dumps({"workload": desc, "affinity": time_affinity(args, wl, pc, ctx, feasible)}), flush=True)
        return
    if only == "delta":
        print(json.dumps({"workload": desc, "rule_delta": time_rule_delta(args, wl, pc, ctx, D)}), flush=True)
        return
    if only == "preferred":
        # the feasible sets are the selector rows' bitsets, computed once
        pc.pc_eval_selectors(D["labels"], D["pred_off"], D["preds"], feasible=feasible, popcnt=popcnt, ctx=ctx)
        torch.cuda.synchronize()
        print(json.dumps({"workload": desc, "preferred": time_preferred(args, wl, pc, ctx, feasible)}), flush=True)
        return
    if only == "update":
        print(json.dumps({"workload": desc, "update": time_update(args, wl, pc, ctx, D, feasible, popcnt)}),
              flush=True)
        return
    if only == "verdict":
        # the inputs the verdict reads, computed once outside the timed pass
        pc.pc_trace_flows(wl["S"], D["port_off"], D["port_peer"], D["jur"], D["rule_off"], D["rules"], D["hdr"],
                          D["ingress"], wl["ttl"], out=traces, ctx=ctx)
        pc.pc_masked_reach(wl["V"], D["adj_off"], D["adj"], D["region"], D["src"], D["allowed"], D["target"],
                           dist=reach, ctx=ctx)
        vo = time_verdict_only(args, wl, pc, ctx, D, traces, reach)
        vo.pop("_pass")
        vo.pop("_reason")
        print(json.dumps({"workload": desc, "verdict_only": vo}), flush=True)
        return
    if only == "synthesis":
        print(json.dumps({"workload": desc, "synthesis": time_synthesis(args, wl, pc, ctx)}), flush=True)
        return
    if only == "paths":
        # the bitsets the verdict reads, computed once outside the timed pass
        pc.pc_eval_selectors(D["labels"], D["pred_off"], D["preds"], feasible=feasible, popcnt=popcnt, ctx=ctx)
        torch.cuda.synchronize()
        print(json.dumps({"workload": desc, "paths": time_paths(args, wl, D, pc, ctx, feasible, popcnt)}), flush=True)
        return

    def step():
        if only in ("all", "sel"):
            pc.pc_eval_selectors(D["labels"], D["pred_off"], D["preds"], feasible=feasible, popcnt=popcnt, ctx=ctx)
        if only in ("all", "trace"):
            pc.pc_trace_flows(wl["S"], D["port_off"], D["port_peer"], D["jur"], D["rule_off"], D["rules"], D["hdr"],
                              D["ingress"], wl["ttl"], out=traces, ctx=ctx)
        if only in ("all", "reach"):
            pc.pc_masked_reach(wl["V"], D["adj_off"], D["adj"], D["region"], D["src"], D["allowed"], D["target"],
                               dist=reach, ctx=ctx)
        if only == "all":
            pc.pc_report(D["intents"], feasible, popcnt, N, traces, D["expect"], reach, pass_=pass_, reason=reason,
                         summary=summary, ctx=ctx)

    elapsed, prof = timed_steps(args, ctx, step)
    flags = ctx.data_errors(clear=True)
    ms_step = 1e3 * elapsed / args.steps

    tr = pc.records(traces, pc.TRACE_OUT_DT)
    ing = wl["ingress"]
    started = (ing >= 0) & (ing < wl["S"])
    lookups = int((tr["hops"][started].astype(np.int64) + 1).sum())
    pairs = int(I_rows) * int(N)
    value = pairs * args.steps / elapsed
    reasons = reason.cpu().numpy() & 0x7F
    passed = int((reasons == 0).sum())

    def ktime(prefix):
        return sum(ms for name, (n, ms) in prof.items() if name.startswith(prefix)) / args.steps

    roof_kernel = "k_sel_eval"
    if only in ("all", "sel"):
        if roof_kernel not in prof:
            raise SystemExit(f"bench: no timing for {roof_kernel} (timed kernels: {sorted(prof)})")
        sel_eval_n, sel_eval_ms = prof[roof_kernel]
    else:
        sel_eval_n, sel_eval_ms = 0, 0.0
    avg_eval_ms = sel_eval_ms / max(sel_eval_n, 1)
    # algorithmic bytes of one launch: the feasible bitsets written, one
    # popcount per row, the node labels and the predicates read once
    n_preds = wl["n_preds"]
    alg_bytes = I_rows * W * 8 + I_rows * 4 + n_preds * 40 + N * L
    achieved = alg_bytes / (avg_eval_ms * 1e-3) / 1e9 if avg_eval_ms > 0 else 0.0
    per_kernel = {name: {"launches_per_step": n / args.steps, "ms_per_step": ms / args.steps}
                  for name, (n, ms) in sorted(prof.items(), key=lambda kv: -kv[1][1])}
    trace_ms = ktime("k_tr_")
    line = {
        "metric": "flow hops traced/sec + selector evals/sec on 1 MI355X; % of peak HBM GB/s",
        "value": value,
        "unit": "selector evals/s ((intent,node) pairs per second of whole-step time)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64 bitsets / int32 (integer work, no floating point)",
        "data": "synthetic (seeded generators; no dataset)",
        "config": {"workload": desc, "intents": I, "selector_rows": I_rows, "nodes": N, "labels": L,
                   "switches": wl["S"], "rules": wl["n_rules"], "traces": T, "reach_queries": Q,
                   "ttl": wl["ttl"], "parallelism": "single GPU"},
        "flow_hops_per_s": lookups * args.steps / elapsed,
        "flow_lookups_per_step": lookups,
        "selector_pairs_per_step": pairs,
        "kernel_rates": {
            "selector_evals_per_s_kernel": pairs / (ktime("k_sel_") * 1e-3) if ktime("k_sel_") else None,
            "flow_hops_per_s_kernel": lookups / (trace_ms * 1e-3) if trace_ms else None,
        },
        "entry_ms_per_step": {"pc_eval_selectors": ktime("k_sel_"), "pc_trace_flows": trace_ms,
                              "pc_masked_reach": ktime("k_rc_"), "pc_report": ktime("k_report")},
        "per_kernel": per_kernel,
        "roofline": {"kernel": roof_kernel, "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": measured_traffic(args.workload, roof_kernel),
                     "alg_bytes_per_launch": alg_bytes, "avg_launch_ms": avg_eval_ms},
        "verdict": {"passed": passed, "intents": I},
        "data_error_flags": flags,
    }
    if only in ("all", "trace") and "k_tr_prep" in prof:
        # rule-table preparation: every 40-byte rule read once, 96 chunk-set
        # words (384 B) written per 32-rule group
        ro = np.asarray(wl["rule_off"], dtype=np.int64)
        groups = int(((np.diff(ro) + 31) // 32).sum())
        prep_bytes = int(wl["n_rules"]) * 40 + groups * 96 * 4
        prep_n, prep_ms = prof["k_tr_prep"]
        prep_avg = prep_ms / max(prep_n, 1)
        prep_gbs = prep_bytes / (prep_avg * 1e-3) / 1e9 if prep_avg > 0 else 0.0
        line["trace_prep_roofline"] = {"kernel": "k_tr_prep", "bound": "hbm", "achieved": prep_gbs,
                                       "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": prep_gbs / HBM_PEAK_GBS,
                                       "traffic": measured_traffic(args.workload, "k_tr_prep"),
                                       "alg_bytes_per_launch": prep_bytes, "avg_launch_ms": prep_avg}
    if only in ("all", "trace"):
        line["trace_roofline"] = trace_roofline(wl, pc, ctx, D, tr, prof, args.steps, args.workload)
    gpu_out = None
    if only == "all" and not args.no_cpu_baseline:
        # the last timed step's outputs, for the oracle's parity check
        gpu_out = {"feasible": feasible.cpu().numpy().view(np.uint64), "popcnt": popcnt.cpu().numpy().view(np.uint32),
                   "traces": tr, "reach": reach.cpu().numpy(), "reason": reason.cpu().numpy()}
    if only == "all" and not args.no_paths:
        line["paths"] = time_paths(args, wl, D, pc, ctx, feasible, popcnt)
    if only == "all" and not args.no_affinity:
        line["affinity"] = time_affinity(args, wl, pc, ctx, feasible)
    if only == "all" and not args.no_preferred:
        line["preferred"] = time_preferred(args, wl, pc, ctx, feasible)
    if only == "all" and not args.no_verdict_only:
        vo = time_verdict_only(args, wl, pc, ctx, D, traces, reach)
        vo["verdict_equals_main_pass"] = bool(torch.equal(vo.pop("_pass"), pass_) and
                                              torch.equal(vo.pop("_reason"), reason))
        vo["main_pass_selector_plus_report_ms"] = ktime("k_sel_") + ktime("k_report")
        line["verdict_only"] = vo
    if only == "all" and not args.no_update:
        line["update"] = time_update(args, wl, pc, ctx, D, feasible, popcnt)
    if only == "all" and not args.no_synthesis:
        line["synthesis"] = time_synthesis(args, wl, pc, ctx)
    if only == "all" and not args.no_rule_delta:
        line["rule_delta"] = time_rule_delta(args, wl, pc, ctx, D)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl, pairs, args.cpu_seconds, gpu=gpu_out)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
