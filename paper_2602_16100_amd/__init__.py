"""MI355X compliance checker -- Python binding of libpc.so.

The library (include/pc.h) runs the validator checks of LLM-driven,
intent-based privacy orchestration (arXiv 2602.16100) as HIP kernels on one
GPU: node-selector evaluation (pc_eval_selectors; full node affinity with
OR-ed terms, six operators and label-inventory flags: pc_eval_affinity), path
synthesis with per-hop rule compilation (pc_synthesize_paths), incremental
re-evaluation after node-label changes and verdict-only runs (pc_update_nodes,
pc_eval_selectors_count, pc_probe_selectors, pc_report_counts), flow-table tracing
(pc_trace_flows), masked reachability (pc_masked_reach) and the per-intent
verdict (pc_report), with waypoint and forbidden-switch constraints
(pc_trace_flows_watch, pc_masked_reach_via, pc_report_paths).

This module only marshals arguments: torch tensors provide device memory
and the current HIP stream; every step of the computation runs in
libpc.so.  There is no CPU fallback -- if the library is missing or no GPU
is present, calls raise.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch  # imported first so that libpc.so binds to the HIP runtime torch already loaded

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "_lib", "libpc.so")

PC_OK, PC_EINVAL, PC_ENOMEM, PC_EDEVICE = 0, -1, -2, -3
PC_EGRESS, PC_DROP, PC_MISS, PC_TTL = 0, 1, 2, 3
DERR = {"PRED": 1, "OFFSETS": 2, "ACTION": 4, "SWITCH": 8, "JUR": 16, "GRAPH": 32, "INTENT": 64, "NODE": 128}

PRED_BYTES, RULE_BYTES, KEY_BYTES, INTENT_BYTES, EXPECT_BYTES = 40, 40, 16, 32, 12
TRACE_OUT_DT = np.dtype([("jmask", "<u4"), ("last_switch", "<i4"), ("last_port", "<u2"),
                         ("hops", "u1"), ("state", "u1")])
SUMMARY_DT = np.dtype([("counts", "<u8", (4, 16)), ("no_path", "<u8", (4,))])
PATH_EXPECT_DT = np.dtype([("must", "<u4"), ("forbid", "<u4")])
RULE_DT = np.dtype([("value", "<u4", (4,)), ("mask", "<u4", (4,)), ("priority", "<u2"), ("action", "<u2"),
                    ("rsv", "<u4")])
SUMMARY_BYTES = 544
assert RULE_DT.itemsize == RULE_BYTES
assert TRACE_OUT_DT.itemsize == 12 and SUMMARY_DT.itemsize == SUMMARY_BYTES and PATH_EXPECT_DT.itemsize == 8


class PCError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"libpc error {code}: {msg}")
        self.code = code


_lib = None


def _hip_runtimes_mapped():
    paths = set()
    try:
        with open("/proc/self/maps") as f:
            for line in f:
                if "libamdhip64" in line:
                    paths.add(os.path.realpath(line.split()[-1]))
    except OSError:
        pass
    return paths


def lib():
    """Load libpc.so once (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: run `python -m paper_2602_16100_amd._build` first")
    L = ctypes.CDLL(LIB_PATH)
    if len(_hip_runtimes_mapped()) > 1:
        raise ImportError(f"two HIP runtimes mapped in this process: {_hip_runtimes_mapped()}")
    P, I32, I64, C = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_int
    L.pc_create.argtypes = [ctypes.POINTER(P), C]
    L.pc_destroy.argtypes = [P]
    L.pc_last_error.argtypes = [P]
    L.pc_last_error.restype = ctypes.c_char_p
    L.pc_version.restype = C
    L.pc_data_errors.argtypes = [P, P, ctypes.POINTER(ctypes.c_uint32), C]
    L.pc_eval_selectors.argtypes = [P, P, I32, I32, P, P, I64, I32, P, P, P]
    L.pc_eval_selectors_noalloc.argtypes = [P, P, I32, I32, P, P, I64, I32, P, P, P]
    L.pc_eval_affinity.argtypes = [P, P, I32, I32, P, I32, P, I32, P, I64, P, P, P, P]
    L.pc_score_preferred.argtypes = [P, P, I32, I32, P, P, I32, P, I32, P, P, I64, P, P, P, P]
    L.pc_update_nodes.argtypes = [P, P, I32, I32, P, P, I64, I32, P, I32, P, P, P]
    L.pc_eval_selectors_count.argtypes = [P, P, I32, I32, P, P, I64, I32, P, P]
    L.pc_probe_selectors.argtypes = [P, P, I32, I32, P, P, I64, I32, P, P, I32, P, P]
    L.pc_report_counts.argtypes = [P, I32, P, I32, P, I32, P, P, I32, P, P, I32, P, P, P, P]
    L.pc_synthesize_paths.argtypes = [P, I32, P, P, I64, P, P, I32, P, P, P, P, I32, P, I32, P, P, I32, I32, P,
                                      P, P, P]
    L.pc_trace_flows.argtypes = [P, I32, P, P, I64, P, P, P, I64, P, P, I32, I32, P, P]
    L.pc_masked_reach.argtypes = [P, I32, P, P, I64, P, I32, P, P, P, P, P]
    L.pc_report.argtypes = [P, I32, P, I32, P, I32, P, I32, P, I32, P, P, I32, P, P, P, P]
    L.pc_trace_flows_watch.argtypes = [P, I32, P, P, I64, P, P, P, I64, P, P, I32, I32, P, I32, P, P, P]
    L.pc_trace_flows_delta.argtypes = [P, I32, P, P, I64, P, P, P, I64, P, P, I32, I32, P, I32, P, P, P, P, P]
    L.pc_masked_reach_via.argtypes = [P, I32, P, P, I64, P, I32, P, P, P, P, I32, P, I32, P, P]
    L.pc_report_paths.argtypes = [P, I32, P, I32, P, I32, P, I32, P, I32, P, P, I32, P, P, P, P, P, P]
    L.pc_trace_keep_tables.argtypes = [P, C]
    L.pc_profile.argtypes = [P, C]
    L.pc_profile_read.argtypes = [P, C, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(I64),
                                  ctypes.POINTER(ctypes.c_double)]
    L.pc_measure_valu.argtypes = [P, C, C, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double), P]
    _lib = L
    return L


EXPORTED = ("pc_create", "pc_destroy", "pc_last_error", "pc_version", "pc_data_errors", "pc_profile",
            "pc_profile_read", "pc_eval_selectors", "pc_eval_affinity", "pc_trace_flows", "pc_masked_reach",
            "pc_report", "pc_trace_flows_watch", "pc_masked_reach_via", "pc_report_paths", "pc_synthesize_paths",
            "pc_update_nodes", "pc_eval_selectors_count", "pc_probe_selectors", "pc_report_counts",
            "pc_score_preferred", "pc_trace_flows_delta", "pc_trace_keep_tables", "pc_eval_selectors_noalloc",
            "pc_measure_valu")


class Context:
    """A libpc context on one device (owns the scratch arena)."""

    def __init__(self, device: int = 0):
        self.device = device
        h = ctypes.c_void_p()
        rc = lib().pc_create(ctypes.byref(h), device)
        if rc != PC_OK:
            raise PCError(rc, f"pc_create(device={device}) failed")
        self.handle = h

    def close(self):
        if self.handle:
            lib().pc_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def check(self, rc):
        if rc != PC_OK:
            raise PCError(rc, lib().pc_last_error(self.handle).decode(errors="replace"))

    def data_errors(self, clear: bool = True, stream=None) -> int:
        """Synchronise the stream and return (and clear) the sticky data-error word."""
        f = ctypes.c_uint32()
        self.check(lib().pc_data_errors(self.handle, _stream(stream), ctypes.byref(f), int(clear)))
        return int(f.value)


    def keep_tables(self, enable: bool):
        """Declare (True) that on this context, consecutive
        pc_trace_flows_delta calls with a change list pass tables that differ
        from the previous call's only in the listed switches: those calls
        then re-prepare only the listed switches.  The library does not check
        unlisted switches, so breaking the promise gives stale results.
        Off by default: every delta call prepares every switch."""
        self.check(lib().pc_trace_keep_tables(self.handle, int(enable)))

    def profile(self, enable: bool):
        """Reset the per-kernel timing tallies and switch timing on or off."""
        self.check(lib().pc_profile(self.handle, int(enable)))

    def measure_valu(self, op: int = 0, reps: int = 10, stream=None) -> tuple:
        """(wave-wide 32-bit integer VALU instructions retired per second,
        shader clock in Hz) for a kernel that does nothing else; op 0 = add /
        sub, 1 = xor, 2 = and-or of three vector sources, 3 = and-or with a
        scalar source, 4 = 64-bit shift, 5 = add / sub in VOP3 encoding, 6 =
        scalar xor, 7 = 64-bit move, 8 = compare into a scalar mask, 9 =
        select by a scalar mask, 10 = bit-field insert, 11 = xor with a scalar
        source, 12 = 32-bit move, 13 = xor with an inline constant, 14 = xor
        with a 32-bit literal (pc_measure_valu)."""
        r = ctypes.c_double()
        c = ctypes.c_double()
        self.check(lib().pc_measure_valu(self.handle, int(op), int(reps), ctypes.byref(r), ctypes.byref(c),
                                         _stream(stream)))
        return float(r.value), float(c.value)

    def profile_read(self) -> dict:
        """{kernel name: (launches, total milliseconds)} since the last reset."""
        out = {}
        i = 0
        while True:
            name = ctypes.c_char_p()
            n = ctypes.c_int64()
            ms = ctypes.c_double()
            rc = lib().pc_profile_read(self.handle, i, ctypes.byref(name), ctypes.byref(n), ctypes.byref(ms))
            if rc != PC_OK:
                break
            out[name.value.decode()] = (int(n.value), float(ms.value))
            i += 1
        return out


_contexts: dict = {}


def context(device: int | None = None) -> Context:
    """The default context of a device (created on first use)."""
    if device is None:
        device = torch.cuda.current_device()
    if device not in _contexts:
        _contexts[device] = Context(device)
    return _contexts[device]


def _ptr(t):
    if t is None:
        return None
    assert t.is_cuda and t.is_contiguous(), "libpc takes contiguous device tensors"
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def to_device(arr: np.ndarray, device="cuda") -> torch.Tensor:
    """A numpy array (plain or a structured record array) as a device tensor.
    Record arrays travel as uint8 [n, record_size]."""
    a = np.ascontiguousarray(arr)
    if a.dtype.fields is not None:
        a = a.view(np.uint8).reshape(arr.shape[0], arr.dtype.itemsize)
    elif a.dtype == np.uint64:
        a = a.view(np.int64)
    elif a.dtype == np.uint32:
        a = a.view(np.int32)
    elif a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(device)


def records(t: torch.Tensor, dtype: np.dtype) -> np.ndarray:
    """Device/host tensor of packed records -> numpy structured array."""
    return t.detach().cpu().contiguous().numpy().view(np.uint8).reshape(-1).view(dtype)


def pc_eval_selectors(labels, pred_off, preds, n_preds=None, feasible=None, popcnt=None, ctx=None, stream=None):
    """A1: feasible-node bitset [I, ceil(N/64)] (int64 storage of uint64 words)
    and popcount [I] (int32 storage of uint32)."""
    ctx = ctx or context()
    N, L = (int(labels.shape[0]), int(labels.shape[1])) if labels.dim() == 2 else (0, 0)
    I = int(pred_off.shape[0]) - 1
    n_preds = int(preds.shape[0]) if n_preds is None else int(n_preds)
    W = (N + 63) // 64
    dev = pred_off.device
    if feasible is None:
        feasible = torch.empty((I, W), dtype=torch.int64, device=dev)
    if popcnt is None:
        popcnt = torch.empty(I, dtype=torch.int32, device=dev)
    ctx.check(lib().pc_eval_selectors(ctx.handle, _ptr(labels) if labels.numel() else None, N, L, _ptr(pred_off),
                                      _ptr(preds) if preds.numel() else None, n_preds, I,
                                      _ptr(feasible) if feasible.numel() else None, _ptr(popcnt), _stream(stream)))
    return feasible, popcnt


def pc_eval_selectors_noalloc(labels, pred_off, preds, feasible, popcnt, n_preds=None, ctx=None, stream=None):
    """pc_eval_selectors into caller-provided feasible [I, ceil(N/64)] and
    popcnt [I] tensors, with no device allocation by the library (its scratch
    is a fixed per-device array of PC_NOALLOC_SCRATCH_BYTES; calls that
    overlap on one device race)."""
    ctx = ctx or context()
    N, L = (int(labels.shape[0]), int(labels.shape[1])) if labels.dim() == 2 else (0, 0)
    I = int(pred_off.shape[0]) - 1
    n_preds = int(preds.shape[0]) if n_preds is None else int(n_preds)
    ctx.check(lib().pc_eval_selectors_noalloc(ctx.handle, _ptr(labels) if labels.numel() else None, N, L,
                                              _ptr(pred_off), _ptr(preds) if preds.numel() else None, n_preds, I,
                                              _ptr(feasible) if feasible.numel() else None, _ptr(popcnt),
                                              _stream(stream)))
    return feasible, popcnt


def pc_eval_affinity(labels, row_off, term_off, preds, n_terms=None, n_preds=None, feasible=None, popcnt=None,
                     unknown=None, ctx=None, stream=None):
    """A1 with full node affinity: rows are ORs of terms (row_off), terms
    ANDs of expressions (term_off, preds; six operators).  Returns the
    feasible-node bitset [I, ceil(N/64)], popcount [I] and the inventory
    flags [I] (uint8: 1 unknown value, 2 unknown label)."""
    ctx = ctx or context()
    N, L = (int(labels.shape[0]), int(labels.shape[1])) if labels.dim() == 2 else (0, 0)
    I = int(row_off.shape[0]) - 1
    n_terms = int(term_off.shape[0]) - 1 if n_terms is None else int(n_terms)
    n_preds = int(preds.shape[0]) if n_preds is None else int(n_preds)
    W = (N + 63) // 64
    dev = row_off.device
    if feasible is None:
        feasible = torch.empty((I, W), dtype=torch.int64, device=dev)
    if popcnt is None:
        popcnt = torch.empty(I, dtype=torch.int32, device=dev)
    if unknown is None:
        unknown = torch.empty(I, dtype=torch.uint8, device=dev)
    ctx.check(lib().pc_eval_affinity(ctx.handle, _ptr(labels) if labels.numel() else None, N, L,
                                     _ptr(row_off), I, _ptr(term_off), n_terms,
                                     _ptr(preds) if preds.numel() else None, n_preds,
                                     _ptr(feasible) if feasible.numel() else None,
                                     _ptr(popcnt) if I else None, _ptr(unknown) if I else None, _stream(stream)))
    return feasible, popcnt, unknown


def pc_score_preferred(labels, row_off, term_off, weight, preds, feasible=None, n_terms=None, n_preds=None,
                       best=None, score=None, count=None, ctx=None, stream=None):
    """A1 preferred node affinity: per row the feasible node of largest summed
    weight of holding terms (lowest index among equals), its score and the
    number of feasible nodes with that score.  feasible: [I, ceil(N/64)]
    int64 storage of the bitset, or None (every node).  Returns (best int32
    [I] (-1: none feasible), score [I] and count [I], int32 storage of
    uint32)."""
    ctx = ctx or context()
    N, L = (int(labels.shape[0]), int(labels.shape[1])) if labels.dim() == 2 else (0, 0)
    I = int(row_off.shape[0]) - 1
    n_terms = int(term_off.shape[0]) - 1 if n_terms is None else int(n_terms)
    n_preds = int(preds.shape[0]) if n_preds is None else int(n_preds)
    dev = row_off.device
    if best is None:
        best = torch.empty(I, dtype=torch.int32, device=dev)
    if score is None:
        score = torch.empty(I, dtype=torch.int32, device=dev)
    if count is None:
        count = torch.empty(I, dtype=torch.int32, device=dev)
    ctx.check(lib().pc_score_preferred(ctx.handle, _ptr(labels) if labels.numel() else None, N, L,
                                       _ptr(feasible) if feasible is not None and feasible.numel() else None,
                                       _ptr(row_off), I, _ptr(term_off), n_terms,
                                       _ptr(weight) if weight.numel() else None,
                                       _ptr(preds) if preds.numel() else None, n_preds,
                                       _ptr(best) if I else None, _ptr(score) if I else None,
                                       _ptr(count) if I else None, _stream(stream)))
    return best, score, count


def pc_eval_selectors_count(labels, pred_off, preds, n_preds=None, popcnt=None, ctx=None, stream=None):
    """NEXT-4: popcount [I] of every selector row, no bitset written."""
    ctx = ctx or context()
    N, L = (int(labels.shape[0]), int(labels.shape[1])) if labels.dim() == 2 else (0, 0)
    I = int(pred_off.shape[0]) - 1
    n_preds = int(preds.shape[0]) if n_preds is None else int(n_preds)
    if popcnt is None:
        popcnt = torch.empty(I, dtype=torch.int32, device=pred_off.device)
    ctx.check(lib().pc_eval_selectors_count(ctx.handle, _ptr(labels) if labels.numel() else None, N, L,
                                            _ptr(pred_off), _ptr(preds) if preds.numel() else None, n_preds, I,
                                            _ptr(popcnt) if I else None, _stream(stream)))
    return popcnt


def pc_probe_selectors(labels, pred_off, preds, probe_row, probe_node, n_preds=None, bits=None, ctx=None,
                       stream=None):
    """NEXT-4: uint8 [P], 1 iff node probe_node[k] satisfies row probe_row[k]."""
    ctx = ctx or context()
    N, L = (int(labels.shape[0]), int(labels.shape[1])) if labels.dim() == 2 else (0, 0)
    I = int(pred_off.shape[0]) - 1
    P = int(probe_row.shape[0])
    n_preds = int(preds.shape[0]) if n_preds is None else int(n_preds)
    if bits is None:
        bits = torch.empty(P, dtype=torch.uint8, device=pred_off.device)
    ctx.check(lib().pc_probe_selectors(ctx.handle, _ptr(labels) if labels.numel() else None, N, L, _ptr(pred_off),
                                       _ptr(preds) if preds.numel() else None, n_preds, I,
                                       _ptr(probe_row) if P else None, _ptr(probe_node) if P else None, P,
                                       _ptr(bits) if P else None, _stream(stream)))
    return bits


def pc_report_counts(intents, popcnt, N, ends, traces, expect, reach, pass_=None, reason=None, summary=None,
                     ctx=None, stream=None):
    """NEXT-4: pc_report from popcounts and per-intent endpoint bits (uint8
    [2I]) instead of the bitset."""
    ctx = ctx or context()
    I = int(intents.shape[0])
    rows = int(popcnt.shape[0])
    T = int(traces.shape[0])
    Q = int(reach.shape[0])
    dev = intents.device
    if pass_ is None:
        pass_ = torch.empty((I + 63) // 64, dtype=torch.int64, device=dev)
    if reason is None:
        reason = torch.empty(I, dtype=torch.uint8, device=dev)
    if summary is None:
        summary = torch.empty(SUMMARY_BYTES, dtype=torch.uint8, device=dev)
    ctx.check(lib().pc_report_counts(ctx.handle, I, _ptr(intents) if I else None, rows, _ptr(popcnt) if rows else None,
                                     int(N), _ptr(ends) if I else None, _ptr(traces) if T else None, T,
                                     _ptr(expect) if I else None, _ptr(reach) if Q else None, Q,
                                     _ptr(pass_) if I else None, _ptr(reason) if I else None, _ptr(summary),
                                     _stream(stream)))
    return pass_, reason, summary


def pc_update_nodes(labels, pred_off, preds, nodes, feasible, popcnt, n_preds=None, ctx=None, stream=None):
    """NEXT-4: re-evaluate every row's bits of the listed nodes (their labels
    changed) in place in feasible / popcnt, which must hold the evaluation
    of the previous labels."""
    ctx = ctx or context()
    N, L = (int(labels.shape[0]), int(labels.shape[1])) if labels.dim() == 2 else (0, 0)
    I = int(pred_off.shape[0]) - 1
    M = int(nodes.shape[0])
    n_preds = int(preds.shape[0]) if n_preds is None else int(n_preds)
    ctx.check(lib().pc_update_nodes(ctx.handle, _ptr(labels) if labels.numel() else None, N, L, _ptr(pred_off),
                                    _ptr(preds) if preds.numel() else None, n_preds, I, _ptr(nodes) if M else None, M,
                                    _ptr(feasible) if feasible.numel() else None, _ptr(popcnt) if I else None,
                                    _stream(stream)))
    return feasible, popcnt


def pc_synthesize_paths(V, port_off, port_peer, region, src, target, allowed, via, forbid, key, out_port, prio,
                        max_hops, weight=None, n_ports=None, hops=None, path=None, rules=None, ctx=None, stream=None):
    """NEXT-2: per request the walk's hop count [Q] (-1 = none), its switches
    [Q, max_hops+1] and one 40-byte rule per switch (uint8 [Q, max_hops+1,
    40]).  via [Q, Kv] / forbid [Q, Kf] int32 (-1 = unused), key [Q, 4]
    uint32 storage, weight int32 storage of uint32 per port or None."""
    ctx = ctx or context()
    Q = int(src.shape[0])
    Kv = int(via.shape[1]) if via.dim() == 2 else 0
    Kf = int(forbid.shape[1]) if forbid.dim() == 2 else 0
    n_ports = int(port_peer.shape[0]) if n_ports is None else int(n_ports)
    dev = src.device
    slots = int(max_hops) + 1
    if hops is None:
        hops = torch.empty(Q, dtype=torch.int32, device=dev)
    if path is None:
        path = torch.empty((Q, slots), dtype=torch.int32, device=dev)
    if rules is None:
        rules = torch.empty((Q, slots, 40), dtype=torch.uint8, device=dev)
    ctx.check(lib().pc_synthesize_paths(ctx.handle, int(V), _ptr(port_off), _ptr(port_peer) if n_ports else None,
                                        n_ports, None if weight is None else _ptr(weight), _ptr(region), Q,
                                        _ptr(src) if Q else None, _ptr(target) if Q else None,
                                        _ptr(allowed) if Q else None, _ptr(via) if Q and Kv else None, Kv,
                                        _ptr(forbid) if Q and Kf else None, Kf, _ptr(key) if Q else None,
                                        _ptr(out_port) if Q else None, int(prio), int(max_hops),
                                        _ptr(hops) if Q else None, _ptr(path) if Q else None,
                                        _ptr(rules) if Q else None, _stream(stream)))
    return hops, path, rules


def pc_trace_flows(S, port_off, port_peer, jur, rule_off, rules, hdr, ingress, ttl, n_ports=None, n_rules=None,
                   out=None, ctx=None, stream=None):
    """A2-A4: one 12-byte pc_trace_out record per trace (uint8 [T, 12])."""
    ctx = ctx or context()
    T = int(ingress.shape[0])
    n_ports = int(port_peer.shape[0]) if n_ports is None else int(n_ports)
    n_rules = int(rules.shape[0]) if n_rules is None else int(n_rules)
    if out is None:
        out = torch.empty((T, 12), dtype=torch.uint8, device=ingress.device)
    ctx.check(lib().pc_trace_flows(ctx.handle, int(S), _ptr(port_off), _ptr(port_peer) if port_peer.numel() else None,
                                   n_ports, _ptr(jur), _ptr(rule_off), _ptr(rules) if rules.numel() else None,
                                   n_rules, _ptr(hdr) if T else None, _ptr(ingress) if T else None, T, int(ttl),
                                   _ptr(out) if T else None, _stream(stream)))
    return out


def pc_masked_reach(V, adj_off, adj, region, src, allowed, target=None, n_adj=None, dist=None, ctx=None,
                    stream=None):
    """A5: BFS hop distances inside the allowed-induced subgraph: [Q, V] when
    target is None, else [Q]; -1 = unreachable."""
    ctx = ctx or context()
    Q = int(src.shape[0])
    n_adj = int(adj.shape[0]) if n_adj is None else int(n_adj)
    if dist is None:
        shape = (Q, int(V)) if target is None else (Q,)
        dist = torch.empty(shape, dtype=torch.int32, device=src.device)
    ctx.check(lib().pc_masked_reach(ctx.handle, int(V), _ptr(adj_off), _ptr(adj) if adj.numel() else None, n_adj,
                                    _ptr(region), Q, _ptr(src) if Q else None, _ptr(allowed) if Q else None,
                                    _ptr(target), _ptr(dist) if dist.numel() else None, _stream(stream)))
    return dist


def pc_report(intents, feasible, popcnt, N, traces, expect, reach, pass_=None, reason=None, summary=None, ctx=None,
              stream=None):
    """A6: pass bits [ceil(I/64)] (int64 storage of uint64), reason codes [I]
    (uint8) and the pc_summary record (uint8 [544])."""
    ctx = ctx or context()
    I = int(intents.shape[0])
    rows = int(feasible.shape[0])
    W = int(feasible.shape[1]) if feasible.dim() == 2 else 0
    T = int(traces.shape[0])
    Q = int(reach.shape[0])
    dev = intents.device
    if pass_ is None:
        pass_ = torch.empty((I + 63) // 64, dtype=torch.int64, device=dev)
    if reason is None:
        reason = torch.empty(I, dtype=torch.uint8, device=dev)
    if summary is None:
        summary = torch.empty(SUMMARY_BYTES, dtype=torch.uint8, device=dev)
    ctx.check(lib().pc_report(ctx.handle, I, _ptr(intents) if I else None, rows,
                              _ptr(feasible) if feasible.numel() else None, W, _ptr(popcnt) if rows else None,
                              int(N), _ptr(traces) if T else None, T, _ptr(expect) if I else None,
                              _ptr(reach) if Q else None, Q, _ptr(pass_) if I else None, _ptr(reason) if I else None,
                              _ptr(summary), _stream(stream)))
    return pass_, reason, summary


def pc_trace_flows_delta(S, port_off, port_peer, jur, rule_off, rules, hdr, ingress, ttl, out, vsum, changed=None,
                         walk=None, n_ports=None, n_rules=None, ctx=None, stream=None):
    """A2+A3 incremental re-trace.  changed=None: trace everything from
    scratch into out (uint8 [T, 12]) and vsum (int64 [T], the visited-switch
    summaries) and, when given, walk (int32 [T, 8], the first 8 switches of
    every walk).  changed = int32 tensor of switch ids: out / vsum / walk
    hold the results on the previous tables; only traces that visited a
    changed switch (exactly, for walks that fit their record; by summary
    bits otherwise) are traced again on the tables given.  Returns the
    number of traces traced again (an int32 device tensor of one element).
    Every switch's tables are prepared again on each call unless the
    context's keep_tables(True) promise is in force (then only the listed
    switches are; the promise is the caller's to keep)."""
    ctx = ctx or context()
    T = int(ingress.shape[0])
    n_ports = int(port_peer.shape[0]) if n_ports is None else int(n_ports)
    n_rules = int(rules.shape[0]) if n_rules is None else int(n_rules)
    C = -1 if changed is None else int(changed.shape[0])
    n = torch.empty(1, dtype=torch.int32, device=ingress.device)
    ctx.check(lib().pc_trace_flows_delta(ctx.handle, int(S), _ptr(port_off), _ptr(port_peer) if n_ports else None,
                                         n_ports, _ptr(jur), _ptr(rule_off), _ptr(rules) if n_rules else None,
                                         n_rules, _ptr(hdr) if T else None, _ptr(ingress) if T else None, T,
                                         int(ttl), _ptr(changed) if C > 0 else None, C, _ptr(out) if T else None,
                                         _ptr(vsum) if T else None, _ptr(walk) if walk is not None and T else None,
                                         _ptr(n), _stream(stream)))
    return n


def pc_trace_flows_watch(S, port_off, port_peer, jur, rule_off, rules, hdr, ingress, ttl, watch, n_ports=None,
                         n_rules=None, out=None, visit=None, ctx=None, stream=None):
    """pc_trace_flows plus, per trace, the visit word over its watch slots:
    watch is int32 [T, K] (K <= 32, -1 = unused); returns (out uint8 [T, 12],
    visit int32 [T] storage of uint32)."""
    ctx = ctx or context()
    T = int(ingress.shape[0])
    K = int(watch.shape[1]) if watch is not None and watch.dim() == 2 else 0
    n_ports = int(port_peer.shape[0]) if n_ports is None else int(n_ports)
    n_rules = int(rules.shape[0]) if n_rules is None else int(n_rules)
    dev = ingress.device
    if out is None:
        out = torch.empty((T, 12), dtype=torch.uint8, device=dev)
    if visit is None:
        visit = torch.empty(T, dtype=torch.int32, device=dev)
    ctx.check(lib().pc_trace_flows_watch(
        ctx.handle, int(S), _ptr(port_off), _ptr(port_peer) if port_peer.numel() else None, n_ports, _ptr(jur),
        _ptr(rule_off), _ptr(rules) if rules.numel() else None, n_rules, _ptr(hdr) if T else None,
        _ptr(ingress) if T else None, T, int(ttl), _ptr(watch) if T and K else None, K, _ptr(out) if T else None,
        _ptr(visit) if T else None, _stream(stream)))
    return out, visit


def pc_masked_reach_via(V, adj_off, adj, region, src, allowed, target, via, forbid, n_adj=None, dist=None, ctx=None,
                        stream=None):
    """Shortest walk through the waypoints via [Q, Kv] avoiding forbid [Q, Kf]
    inside the allowed-induced subgraph: int32 [Q], -1 = none."""
    ctx = ctx or context()
    Q = int(src.shape[0])
    Kv = int(via.shape[1]) if via is not None and via.dim() == 2 else 0
    Kf = int(forbid.shape[1]) if forbid is not None and forbid.dim() == 2 else 0
    n_adj = int(adj.shape[0]) if n_adj is None else int(n_adj)
    if dist is None:
        dist = torch.empty(Q, dtype=torch.int32, device=src.device)
    ctx.check(lib().pc_masked_reach_via(
        ctx.handle, int(V), _ptr(adj_off), _ptr(adj) if adj.numel() else None, n_adj, _ptr(region), Q,
        _ptr(src) if Q else None, _ptr(allowed) if Q else None, _ptr(target) if Q else None,
        _ptr(via) if Q and Kv else None, Kv, _ptr(forbid) if Q and Kf else None, Kf, _ptr(dist) if Q else None,
        _stream(stream)))
    return dist


def pc_report_paths(intents, feasible, popcnt, N, traces, expect, reach, visit, pexp, pass_=None, reason=None,
                    summary=None, ctx=None, stream=None):
    """pc_report with the forbidden-switch and waypoint checks: visit [T]
    (from pc_trace_flows_watch) and pexp, pc_path_expect records (uint8
    [I, 8])."""
    ctx = ctx or context()
    I = int(intents.shape[0])
    rows = int(feasible.shape[0])
    W = int(feasible.shape[1]) if feasible.dim() == 2 else 0
    T = int(traces.shape[0])
    Q = int(reach.shape[0])
    dev = intents.device
    if pass_ is None:
        pass_ = torch.empty((I + 63) // 64, dtype=torch.int64, device=dev)
    if reason is None:
        reason = torch.empty(I, dtype=torch.uint8, device=dev)
    if summary is None:
        summary = torch.empty(SUMMARY_BYTES, dtype=torch.uint8, device=dev)
    ctx.check(lib().pc_report_paths(
        ctx.handle, I, _ptr(intents) if I else None, rows, _ptr(feasible) if feasible.numel() else None, W,
        _ptr(popcnt) if rows else None, int(N), _ptr(traces) if T else None, T, _ptr(expect) if I else None,
        _ptr(reach) if Q else None, Q, _ptr(visit) if T else None, _ptr(pexp) if I else None,
        _ptr(pass_) if I else None, _ptr(reason) if I else None, _ptr(summary), _stream(stream)))
    return pass_, reason, summary


def version() -> int:
    return int(lib().pc_version())
