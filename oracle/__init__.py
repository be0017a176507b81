"""CPU oracle for the compliance check -- TEST INFRASTRUCTURE.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package.  It wraps `pc_oracle.c` (plain C loops, OpenMP over
the outermost loop only) through ctypes.  It shares nothing with the GPU
library: its own record layouts, its own build, its own loops.

Each function states the passage of the paper it follows in the C source.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pc_oracle.c")
# PC_ORACLE_LIB names another build of the same source (the sanitizer test
# loads an AddressSanitizer / UBSan build through it)
_LIB = os.environ.get("PC_ORACLE_LIB") or os.path.join(_HERE, "_pc_oracle.so")

TRACE_DT = np.dtype([("jmask", "<u4"), ("last_switch", "<i4"), ("last_port", "<u2"),
                     ("hops", "u1"), ("state", "u1")])
assert TRACE_DT.itemsize == 12
SUMMARY_DT = np.dtype([("counts", "<u8", (4, 16)), ("no_path", "<u8", (4,))])
PATH_EXPECT_DT = np.dtype([("must", "<u4"), ("forbid", "<u4")])
RULE_DT = np.dtype([("value", "<u4", (4,)), ("mask", "<u4", (4,)), ("priority", "<u2"), ("action", "<u2"),
                    ("rsv", "<u4")])
assert RULE_DT.itemsize == 40

EGRESS, DROP, MISS, TTL = 0, 1, 2, 3
F_PRED, F_OFFSETS, F_ACTION, F_SWITCH, F_JUR, F_GRAPH, F_INTENT, F_NODE = 1, 2, 4, 8, 16, 32, 64, 128

_lib = None


def build(force=True, out=None, sanitize=False):
    """Compile the oracle with gcc (-O2, OpenMP).  sanitize=True adds
    AddressSanitizer and UBSan (every finding aborts) for a build at `out`."""
    out = out or _LIB
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Werror"]
    if sanitize:
        cmd += ["-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]
    cmd += ["-o", out + ".tmp", _SRC]
    if force or not os.path.exists(out):
        subprocess.check_call(cmd)
        os.replace(out + ".tmp", out)
    return out


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        _lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        I64 = ctypes.c_int64
        C = ctypes.c_int
        _lib.orc_selectors.argtypes = [P, I64, I64, P, P, I64, I64, P, I64, P, P, P, C]
        _lib.orc_affinity.argtypes = [P, I64, I64, P, I64, P, I64, P, I64, P, I64, P, P, P, P, C]
        _lib.orc_preferred.argtypes = [P, I64, I64, P, P, I64, P, I64, P, P, I64, P, I64, P, P, P, P, C]
        _lib.orc_update_nodes.argtypes = [P, I64, I64, P, P, I64, I64, P, I64, P, P, P, C]
        _lib.orc_probes.argtypes = [P, I64, I64, P, P, I64, I64, P, P, I64, P, P]
        _lib.orc_synthesize.argtypes = [I64, P, P, I64, P, P, I64, P, P, P, P, I64, P, I64, P, P, I64, I64, P,
                                        I64, P, P, P, P, C]
        _lib.orc_trace.argtypes = [I64, P, P, I64, P, P, P, I64, P, P, I64, I64, P, I64, P, I64, P, P, P, P, P, C]
        _lib.orc_reach.argtypes = [I64, P, P, I64, P, I64, P, P, P, P, I64, P, P, C]
        _lib.orc_reach_via.argtypes = [I64, P, P, I64, P, I64, P, P, P, P, I64, P, I64, P, I64, P, P, C]
        _lib.orc_report.argtypes = [I64, P, I64, P, I64, P, I64, P, I64, P, P, I64, P, P, P, P, P, P]
        _lib.orc_max_threads.restype = C
    return _lib


def _p(a):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def max_threads():
    return int(_load().orc_max_threads())


def selectors(labels, pred_off, preds, n_preds=None, rows=None, nthreads=0):
    """Feasible-node bitset and popcount for the given selector rows
    (all rows by default).  Returns (feasible [nrows, W] u64, popcnt u32, flags)."""
    lib = _load()
    labels = np.ascontiguousarray(labels, np.uint8)
    N, L = labels.shape
    I = pred_off.shape[0] - 1
    if rows is None:
        rows = np.arange(I, dtype=np.int32)
    rows = np.ascontiguousarray(rows, np.int32)
    n_preds = preds.shape[0] if n_preds is None else n_preds
    W = (N + 63) // 64
    feas = np.zeros((rows.shape[0], W), np.uint64)
    pc = np.zeros(rows.shape[0], np.uint32)
    err = np.zeros(1, np.uint32)
    lib.orc_selectors(_p(labels), N, L, _p(np.ascontiguousarray(pred_off, np.int32)),
                      _p(np.ascontiguousarray(preds)), n_preds, I, _p(rows), rows.shape[0],
                      _p(feas), _p(pc), _p(err), nthreads)
    return feas, pc, int(err[0])


def update_nodes(labels, pred_off, preds, nodes, feasible, popcnt, n_preds=None, nthreads=0):
    """Incremental re-evaluation after the labels of `nodes` changed: returns
    (feasible', popcnt', flags) from copies of the given feasible [I, W] and
    popcnt [I] (which must hold the evaluation on the previous labels)."""
    lib = _load()
    labels = np.ascontiguousarray(labels, np.uint8)
    N, L = labels.shape
    I = pred_off.shape[0] - 1
    n_preds = preds.shape[0] if n_preds is None else n_preds
    f = np.array(feasible, np.uint64, copy=True, order="C")
    pc = np.array(popcnt, np.uint32, copy=True)
    nodes = np.ascontiguousarray(nodes, np.int32)
    err = np.zeros(1, np.uint32)
    lib.orc_update_nodes(_p(labels), N, L, _p(np.ascontiguousarray(pred_off, np.int32)), _p(np.ascontiguousarray(preds)),
                         n_preds, I, _p(nodes), nodes.shape[0], _p(f), _p(pc), _p(err), nthreads)
    return f, pc, int(err[0])


def probes(labels, pred_off, preds, probe_row, probe_node, n_preds=None):
    """bit[k] = node probe_node[k] satisfies selector row probe_row[k]
    (0 when either is out of range).  Returns (bits u8, flags)."""
    lib = _load()
    labels = np.ascontiguousarray(labels, np.uint8)
    N, L = labels.shape
    I = pred_off.shape[0] - 1
    n_preds = preds.shape[0] if n_preds is None else n_preds
    pr = np.ascontiguousarray(probe_row, np.int32)
    pn = np.ascontiguousarray(probe_node, np.int32)
    bits = np.zeros(pr.shape[0], np.uint8)
    err = np.zeros(1, np.uint32)
    lib.orc_probes(_p(labels), N, L, _p(np.ascontiguousarray(pred_off, np.int32)), _p(np.ascontiguousarray(preds)),
                   n_preds, I, _p(pr), _p(pn), pr.shape[0], _p(bits), _p(err))
    return bits, int(err[0])


def affinity(labels, row_off, term_off, preds, n_terms=None, n_preds=None, rows=None, nthreads=0):
    """Required node affinity: rows are ORs of terms, terms ANDs of
    expressions (six operators).  Returns (feasible [nrows, W] u64,
    popcnt u32, unknown u8 (bit 0 unknown value, bit 1 unknown label),
    flags)."""
    lib = _load()
    labels = np.ascontiguousarray(labels, np.uint8)
    N, L = labels.shape
    I = row_off.shape[0] - 1
    n_terms = term_off.shape[0] - 1 if n_terms is None else n_terms
    n_preds = preds.shape[0] if n_preds is None else n_preds
    if rows is None:
        rows = np.arange(I, dtype=np.int32)
    rows = np.ascontiguousarray(rows, np.int32)
    W = (N + 63) // 64
    feas = np.zeros((rows.shape[0], W), np.uint64)
    pc = np.zeros(rows.shape[0], np.uint32)
    unk = np.zeros(rows.shape[0], np.uint8)
    err = np.zeros(1, np.uint32)
    lib.orc_affinity(_p(labels), N, L, _p(np.ascontiguousarray(row_off, np.int32)), I,
                     _p(np.ascontiguousarray(term_off, np.int32)), n_terms, _p(np.ascontiguousarray(preds)),
                     n_preds, _p(rows), rows.shape[0], _p(feas), _p(pc), _p(unk), _p(err), nthreads)
    return feas, pc, unk, int(err[0])


def preferred(labels, row_off, term_off, weight, preds, feasible=None, n_terms=None, n_preds=None, rows=None,
              nthreads=0):
    """Preferred node affinity: per row the feasible node of largest summed
    weight of holding terms (lowest index among equals; -1 when no node is
    feasible), that score and the number of feasible nodes reaching it.
    feasible: [I, W] u64 bitset or None (every node).  Returns (best int32,
    score u32, count u32, flags)."""
    lib = _load()
    labels = np.ascontiguousarray(labels, np.uint8)
    N, L = labels.shape
    I = row_off.shape[0] - 1
    n_terms = term_off.shape[0] - 1 if n_terms is None else n_terms
    n_preds = preds.shape[0] if n_preds is None else n_preds
    if rows is None:
        rows = np.arange(I, dtype=np.int32)
    rows = np.ascontiguousarray(rows, np.int32)
    nr = rows.shape[0]
    best = np.zeros(nr, np.int32)
    score = np.zeros(nr, np.uint32)
    count = np.zeros(nr, np.uint32)
    err = np.zeros(1, np.uint32)
    fz = None if feasible is None else np.ascontiguousarray(feasible, np.uint64)
    lib.orc_preferred(_p(labels), N, L, None if fz is None else _p(fz), _p(np.ascontiguousarray(row_off, np.int32)),
                      I, _p(np.ascontiguousarray(term_off, np.int32)), n_terms,
                      _p(np.ascontiguousarray(weight, np.uint32)), _p(np.ascontiguousarray(preds)), n_preds,
                      _p(rows), nr, _p(best), _p(score), _p(count), _p(err), nthreads)
    return best, score, count, int(err[0])


def synthesize(V, port_off, port_peer, region, src, target, allowed, via, forbid, key, out_port, prio, max_hops,
               weight=None, qidx=None, n_ports=None, nthreads=0):
    """Path synthesis: per request the walk's hop count (-1 = none), its
    switches [nq, max_hops+1] (-1 past the end) and one rule per switch
    [nq, max_hops+1] (zero past the end).  via [Q, Kv] / forbid [Q, Kf]
    switch ids, -1 = unused; key uint32 [Q, 4]; weight uint32 per port or
    None (every link weighs 1).  Returns (hops, path, rules, flags)."""
    lib = _load()
    Q = src.shape[0]
    if qidx is None:
        qidx = np.arange(Q, dtype=np.int64)
    qidx = np.ascontiguousarray(qidx, np.int64)
    via = np.ascontiguousarray(via, np.int32)
    via = via.reshape(Q, via.shape[1] if via.ndim == 2 else 1)
    forbid = np.ascontiguousarray(forbid, np.int32)
    forbid = forbid.reshape(Q, forbid.shape[1] if forbid.ndim == 2 else 1)
    n_ports = port_peer.shape[0] if n_ports is None else n_ports
    slots = max_hops + 1
    hops = np.zeros(qidx.shape[0], np.int32)
    path = np.zeros((qidx.shape[0], slots), np.int32)
    rules = np.zeros((qidx.shape[0], slots), RULE_DT)
    err = np.zeros(1, np.uint32)
    lib.orc_synthesize(V, _p(np.ascontiguousarray(port_off, np.int32)), _p(np.ascontiguousarray(port_peer, np.int32)),
                       n_ports, None if weight is None else _p(np.ascontiguousarray(weight, np.uint32)),
                       _p(np.ascontiguousarray(region, np.uint8)), Q, _p(np.ascontiguousarray(src, np.int32)),
                       _p(np.ascontiguousarray(target, np.int32)), _p(np.ascontiguousarray(allowed, np.uint32)),
                       _p(via), via.shape[1], _p(forbid), forbid.shape[1],
                       _p(np.ascontiguousarray(key, np.uint32)), _p(np.ascontiguousarray(out_port, np.int32)),
                       int(prio), int(max_hops), _p(qidx), qidx.shape[0], _p(hops), _p(path), _p(rules), _p(err),
                       nthreads)
    return hops, path, rules, int(err[0])


def trace(S, port_off, port_peer, jur, rule_off, rules, hdr, ingress, ttl, idx=None,
          n_ports=None, n_rules=None, nthreads=0, watch=None, summary=False):
    """Trace records for the given trace indices (all by default).  With a
    watch list [T, K] (switch ids, -1 = unused) also returns the visit words,
    with summary=True the visited-switch summaries (u64, bit s mod 64) and
    the walk records (int32 [n, 8], the first 8 switches, -1 past the end):
    (out, [visit,] [vsum, walk,] flags)."""
    lib = _load()
    T = ingress.shape[0]
    if idx is None:
        idx = np.arange(T, dtype=np.int64)
    idx = np.ascontiguousarray(idx, np.int64)
    out = np.zeros(idx.shape[0], TRACE_DT)
    err = np.zeros(1, np.uint32)
    K = 0
    visit = None
    if watch is not None:
        watch = np.ascontiguousarray(watch, np.int32)
        assert watch.ndim == 2 and watch.shape[0] == T
        K = watch.shape[1]
        visit = np.zeros(idx.shape[0], np.uint32)
    vsum = np.zeros(idx.shape[0], np.uint64) if summary else None
    walk = np.zeros((idx.shape[0], 8), np.int32) if summary else None
    n_ports = port_peer.shape[0] if n_ports is None else n_ports
    n_rules = rules.shape[0] if n_rules is None else n_rules
    lib.orc_trace(S, _p(np.ascontiguousarray(port_off, np.int32)),
                  _p(np.ascontiguousarray(port_peer, np.int32)), n_ports,
                  _p(np.ascontiguousarray(jur, np.uint8)), _p(np.ascontiguousarray(rule_off, np.int32)),
                  _p(np.ascontiguousarray(rules)), n_rules,
                  _p(np.ascontiguousarray(hdr, np.uint32)), _p(np.ascontiguousarray(ingress, np.int32)),
                  T, ttl, _p(watch), K, _p(idx), idx.shape[0], _p(out), _p(visit), _p(vsum), _p(walk), _p(err),
                  nthreads)
    res = [out]
    if watch is not None:
        res.append(visit)
    if summary:
        res.append(vsum)
        res.append(walk)
    res.append(int(err[0]))
    return tuple(res)


def reach(V, adj_off, adj, region, src, allowed, target=None, qidx=None, n_adj=None, nthreads=0):
    """Masked BFS distances: full rows [nq, V] when target is None, else [nq]."""
    lib = _load()
    Q = src.shape[0]
    if qidx is None:
        qidx = np.arange(Q, dtype=np.int64)
    qidx = np.ascontiguousarray(qidx, np.int64)
    n_adj = adj.shape[0] if n_adj is None else n_adj
    if target is None:
        dist = np.zeros((qidx.shape[0], V), np.int32)
    else:
        dist = np.zeros(qidx.shape[0], np.int32)
        target = np.ascontiguousarray(target, np.int32)
    assert target is None or target.shape[0] == Q
    err = np.zeros(1, np.uint32)
    lib.orc_reach(V, _p(np.ascontiguousarray(adj_off, np.int32)), _p(np.ascontiguousarray(adj, np.int32)),
                  n_adj, _p(np.ascontiguousarray(region, np.uint8)), Q, _p(np.ascontiguousarray(src, np.int32)),
                  _p(np.ascontiguousarray(allowed, np.uint32)), _p(target), _p(qidx), qidx.shape[0],
                  _p(dist), _p(err), nthreads)
    return dist, int(err[0])


def reach_via(V, adj_off, adj, region, src, allowed, target, via, forbid, qidx=None, n_adj=None, nthreads=0):
    """Shortest walk src -> via... -> target over allowed, non-forbidden
    vertices: int32 [nq], -1 = none.  via [Q, Kv] and forbid [Q, Kf] hold
    vertex ids, -1 = unused (via ends at its first -1)."""
    lib = _load()
    Q = src.shape[0]
    if qidx is None:
        qidx = np.arange(Q, dtype=np.int64)
    qidx = np.ascontiguousarray(qidx, np.int64)
    n_adj = adj.shape[0] if n_adj is None else n_adj
    via = np.ascontiguousarray(via, np.int32)
    forbid = np.ascontiguousarray(forbid, np.int32)
    assert via.ndim == 2 and forbid.ndim == 2 and via.shape[0] == Q and forbid.shape[0] == Q
    dist = np.zeros(qidx.shape[0], np.int32)
    err = np.zeros(1, np.uint32)
    lib.orc_reach_via(V, _p(np.ascontiguousarray(adj_off, np.int32)), _p(np.ascontiguousarray(adj, np.int32)),
                      n_adj, _p(np.ascontiguousarray(region, np.uint8)), Q, _p(np.ascontiguousarray(src, np.int32)),
                      _p(np.ascontiguousarray(allowed, np.uint32)), _p(np.ascontiguousarray(target, np.int32)),
                      _p(via), via.shape[1], _p(forbid), forbid.shape[1], _p(qidx), qidx.shape[0], _p(dist),
                      _p(err), nthreads)
    return dist, int(err[0])


def report(intents, feasible, popcnt, N, traces, expect, reach_d, visit=None, pexp=None):
    """Per-intent pass bits, reason codes and the (kind, reason) summary.
    With visit words [T] and path expectations [I] (PATH_EXPECT_DT) the
    forbidden-switch and waypoint checks are added."""
    lib = _load()
    I = intents.shape[0]
    feasible = np.ascontiguousarray(feasible, np.uint64)
    rows = feasible.shape[0]
    W = feasible.shape[1] if feasible.ndim == 2 else 0
    traces = np.ascontiguousarray(traces)
    reach_d = np.ascontiguousarray(reach_d, np.int32)
    pass_ = np.zeros((I + 63) // 64, np.uint64)
    reason = np.zeros(I, np.uint8)
    summ = np.zeros(1, SUMMARY_DT)
    err = np.zeros(1, np.uint32)
    lib.orc_report(I, _p(np.ascontiguousarray(intents)), rows, _p(feasible), W,
                   _p(np.ascontiguousarray(popcnt, np.uint32)), N, _p(traces), traces.shape[0],
                   _p(np.ascontiguousarray(expect)), _p(reach_d), reach_d.shape[0],
                   _p(None if visit is None else np.ascontiguousarray(visit, np.uint32)),
                   _p(None if pexp is None else np.ascontiguousarray(pexp)),
                   _p(pass_), _p(reason), _p(summ), _p(err))
    return pass_, reason, summ[0], int(err[0])


def run_workload(wl, nthreads=0):
    """All four stages of a synth.Workload on the CPU (small workloads)."""
    out = {}
    if "labels" in wl.arrays:
        out["feasible"], out["popcnt"], out["sel_err"] = selectors(
            wl["labels"], wl["pred_off"], wl["preds"], nthreads=nthreads)
    if "rules" in wl.arrays:
        out["traces"], out["trace_err"] = trace(
            wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"], wl["rules"],
            wl["hdr"], wl["ingress"], wl["ttl"], nthreads=nthreads)
    if "src" in wl.arrays:
        out["reach"], out["reach_err"] = reach(
            wl["V"], wl["adj_off"], wl["adj"], wl["region"], wl["src"], wl["allowed"],
            wl.arrays.get("target"), nthreads=nthreads)
    if "intents" in wl.arrays:
        out["pass"], out["reason"], out["summary"], out["report_err"] = report(
            wl["intents"], out["feasible"], out["popcnt"], wl["N"], out["traces"], wl["expect"],
            out["reach"])
    return out
