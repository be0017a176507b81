"""Pins for the oracle's per-intent verdict.

Pins: the paper's failure modes as fixtures (transit switch in another
region -> leak with no compliant path; a network policy with no concrete
flow -> no-op, not enforced; a hallucinated label -> no feasible node),
closed forms (a compute-only intent passes iff its row admits a node; a
passing network intent has a compliant path no longer than its trace),
and the summary as the histogram of reasons.
"""
import numpy as np
import pytest

import synth
from helpers import leak_fixture as _leak_fixture, load_golden

REASONS = {"PASS": 0, "NO_FEASIBLE_NODE": 1, "ENDPOINT_INFEASIBLE": 2, "NO_FLOW": 3, "LEAK": 4,
           "UNDELIVERED": 5, "WRONG_EGRESS": 6, "MALFORMED": 7}


def test_paper_transit_leak_and_noop(orc):
    fx, topo, path, key, rule_off, rules = _leak_fixture()
    S = topo["S"]
    tr, err = orc.trace(S, topo["port_off"], topo["port_peer"], topo["jur"], rule_off, rules,
                        key[None, :], np.array([path[0]], np.int32), 16)
    assert err == 0 and tr[0]["state"] == orc.EGRESS and tr[0]["hops"] == 2
    cases = fx["intents"]
    I = len(cases)
    intents = np.zeros(I, synth.INTENT_DT)
    expect = np.zeros(I, synth.EXPECT_DT)
    allowed = np.zeros(I, np.uint32)
    for i, c in enumerate(cases):
        allowed[i] = sum(1 << fx["regions"].index(r) for r in c["allowed"])
        intents[i]["kind"] = synth.KIND_NETWORK
        intents[i]["sel_row"] = -1
        intents[i]["trace_begin"] = 0
        intents[i]["trace_end"] = c["flows"]
        intents[i]["allowed"] = allowed[i]
        expect[i] = (path[-1], len(topo["nbr"][path[-1]]), i if c["flows"] else -1)
    reach, _ = orc.reach(S, topo["adj_off"], topo["adj"], topo["jur"], np.full(I, path[0], np.int32),
                         allowed, np.full(I, path[-1], np.int32))
    feas = np.zeros((0, 1), np.uint64)
    pss, reason, summ, err = orc.report(intents, feas, np.zeros(0, np.uint32), 0, tr, expect, reach)
    assert err == 0
    for i, c in enumerate(cases):
        assert reason[i] & 0x7F == REASONS[c["expect_reason"]], c["cite"]
        if "expect_no_path" in c:
            assert bool(reason[i] & 0x80) == c["expect_no_path"]
        if "expect_reach" in c:
            assert reach[i] == c["expect_reach"]
        assert bool((int(pss[0]) >> i) & 1) == (c["expect_reason"] == "PASS")


def test_paper_hallucinated_label_fails_closed(orc):
    """A compute intent whose selector names a label value no node carries
    has an empty feasible set: NO_FEASIBLE_NODE."""
    from helpers import encode_label_matrix, encode_selector
    fx = load_golden("paper_label_matrix.json")
    labels, vocab = encode_label_matrix(fx)
    preds = encode_selector(fx, vocab, [["region", "In", ["eu_region"]]])
    preds2 = encode_selector(fx, vocab, [["security", "In", ["high"]], ["zone", "In", ["cloud"]]])
    allp = np.concatenate([preds, preds2])
    off = np.array([0, 1, 3], np.int32)
    feas, pc, _ = orc.selectors(labels, off, allp)
    intents = np.zeros(3, synth.INTENT_DT)
    intents["kind"] = [synth.KIND_COMPUTE, synth.KIND_COMPUTE, synth.KIND_HYBRID]
    intents["sel_row"] = [0, 1, 1]
    intents["src_node"] = [-1, -1, 3]      # worker-4 (feasible) ...
    intents["dst_node"] = [-1, -1, 0]      # ... and worker-1 (edge zone: infeasible)
    intents["trace_begin"] = 0
    intents["trace_end"] = [0, 0, 1]
    expect = np.zeros(3, synth.EXPECT_DT)
    expect["dst_switch"] = -1
    expect["dst_port"] = -1
    expect["reach_q"] = -1
    tr = np.zeros(1, orc.TRACE_DT)
    pss, reason, summ, err = orc.report(intents, feas, pc, labels.shape[0], tr, expect, np.zeros(0, np.int32))
    assert list(reason) == [1, 0, 2]
    assert int(pss[0]) == 0b010


def _check_invariants(orc, wl, out):
    it, ex = wl["intents"], wl["expect"]
    reason, pss, summ = out["reason"], out["pass"], out["summary"]
    I = it.shape[0]
    bits = np.array([(int(pss[i >> 6]) >> (i & 63)) & 1 for i in range(I)])
    assert np.array_equal(bits == 1, (reason & 0x7F) == 0)
    # summary = histogram of reasons per kind
    hist = np.zeros((4, 16), np.uint64)
    np.add.at(hist, (it["kind"] & 3, reason & 0x7F), 1)
    assert np.array_equal(summ["counts"], hist)
    nop = np.zeros(4, np.uint64)
    np.add.at(nop, it["kind"] & 3, (reason >> 7).astype(np.uint64))
    assert np.array_equal(summ["no_path"], nop)
    # compute-only: pass iff the row admits a node
    c = np.flatnonzero(it["kind"] == synth.KIND_COMPUTE)
    assert np.array_equal(bits[c] == 1, out["popcnt"][it["sel_row"][c]] > 0)
    # a passing network intent has a compliant path no longer than its trace
    for i in np.flatnonzero((it["kind"] & 2) != 0):
        if bits[i]:
            q = ex["reach_q"][i]
            d = out["reach"][q]
            for t in range(it["trace_begin"][i], it["trace_end"][i]):
                assert 0 <= d <= out["traces"][t]["hops"]
                # a passing network intent's traces stay inside its allowed jurisdictions
                assert int(out["traces"][t]["jmask"]) & ~int(it["allowed"][i]) == 0
                assert out["traces"][t]["state"] == orc.EGRESS
            assert reason[i] & 0x80 == 0
    # the padding bits of the pass vector are zero
    if I % 64:
        assert int(pss[-1]) >> (I % 64) == 0


def test_cfg1_end_to_end_invariants(orc):
    wl = synth.cfg1(0)
    out = orc.run_workload(wl)
    _check_invariants(orc, wl, out)
    # every reason class the tiny case can produce shows up
    assert set(np.unique(out["reason"] & 0x7F)) >= {0, 1, 4}


def test_combined_small_invariants(orc):
    wl = synth.combined_workload(13, 2000, 16, 8, 4, 256, 1501)
    out = orc.run_workload(wl)
    _check_invariants(orc, wl, out)
    r = out["reason"] & 0x7F
    assert (r == 0).sum() > 100 and (r == 4).sum() > 50 and (r == 5).sum() > 20


@pytest.mark.parametrize("field,value", [("kind", 0), ("kind", 4), ("sel_row", 99), ("src_node", 16),
                                         ("trace_end", 5000), ("trace_begin", -1)])
def test_malformed_intent(orc, field, value):
    wl = synth.cfg1(0)
    out = orc.run_workload(wl)
    it = wl["intents"].copy()
    i = 2                                           # a hybrid intent
    it[i][field] = value
    pss, reason, summ, err = orc.report(it, out["feasible"], out["popcnt"], wl["N"], out["traces"],
                                        wl["expect"], out["reach"])
    assert reason[i] == 7 and err & orc.F_INTENT


# ---------------------------------------------------------------------------
# Hand-derived verdict cases (validator check definition: an intent passes
# only if every check passes; the reading orders the failure codes
# NO_FEASIBLE_NODE < ENDPOINT_INFEASIBLE < NO_FLOW < LEAK < UNDELIVERED <
# WRONG_EGRESS, and an intent's reason is the smallest code over its checks).
# Each trace record is written by hand: (jmask, last_switch, last_port, hops,
# state).  The expected reason is worked out from that reading alone.
# ---------------------------------------------------------------------------

E, D, M, T = 0, 1, 2, 3          # EGRESS, DROP, MISS, TTL

# (name, allowed, dst_switch, dst_port, [traces], expected reason)
_NET_CASES = [
    ("all good", 0b0011, 5, 2, [(0b0011, 5, 2, 3, E)], 0),
    ("leak then undelivered", 0b0011, 5, 2, [(0b0111, 5, 2, 3, E), (0b0001, 4, 0xFFFF, 1, D)], 4),
    ("undelivered then leak", 0b0011, 5, 2, [(0b0001, 4, 0xFFFF, 1, M), (0b0111, 5, 2, 3, E)], 4),
    ("wrong egress then undelivered", 0b0011, 5, 2, [(0b0011, 6, 2, 3, E), (0b0001, 4, 0xFFFF, 2, T)], 5),
    ("undelivered then wrong egress", 0b0011, 5, 2, [(0b0001, 4, 0xFFFF, 2, T), (0b0011, 5, 1, 3, E)], 5),
    ("wrong egress after a pass", 0b0011, 5, 2, [(0b0011, 5, 2, 3, E), (0b0011, 5, 3, 3, E)], 6),
    ("leak after a pass", 0b0011, 5, 2, [(0b0011, 5, 2, 3, E), (0b1001, 5, 2, 3, E)], 4),
    ("wrong switch, right port", 0b0011, 5, 2, [(0b0011, 7, 2, 3, E)], 6),
    ("right switch, wrong port", 0b0011, 5, 2, [(0b0011, 5, 0, 3, E)], 6),
    ("any switch, wrong port", 0b0011, -1, 2, [(0b0011, 9, 1, 3, E)], 6),
    ("wrong switch, any port", 0b0011, 5, -1, [(0b0011, 8, 1, 3, E)], 6),
    ("any switch and port", 0b0011, -1, -1, [(0b0011, 8, 1, 3, E)], 0),
    ("drop is undelivered", 0b0011, 5, 2, [(0b0011, 5, 0xFFFF, 3, D)], 5),
    ("ttl is undelivered", 0b0011, 5, 2, [(0b0011, 5, 0xFFFF, 3, T)], 5),
    ("miss is undelivered", 0b0011, 5, 2, [(0b0011, 5, 0xFFFF, 3, M)], 5),
    ("leak beats wrong egress", 0b0011, 5, 2, [(0b0011, 5, 1, 3, E), (0b0110, 6, 2, 3, E)], 4),
    ("no flow", 0b0011, 5, 2, [], 3),
]
# A leak into each jurisdiction bit, one at a time; bits 0 and 31 included.
for _b in (0, 1, 2, 7, 16, 30, 31):
    _allowed = 0xFFFFFFFF & ~(1 << _b)
    _NET_CASES.append((f"leak into jurisdiction {_b}", _allowed, 5, 2,
                       [((1 << _b) | (1 << ((_b + 5) % 32)), 5, 2, 3, E)], 4))
    _NET_CASES.append((f"jurisdiction {_b} allowed", 0xFFFFFFFF, 5, 2,
                       [((1 << _b) | (1 << ((_b + 5) % 32)), 5, 2, 3, E)], 0))


def _net_case_arrays(cases, kind=synth.KIND_NETWORK, sel_row=-1, src_node=-1, dst_node=-1):
    I = len(cases)
    intents = np.zeros(I, synth.INTENT_DT)
    expect = np.zeros(I, synth.EXPECT_DT)
    trs = []
    for i, (_, allowed, dsw, dport, tl, _) in enumerate(cases):
        intents[i]["kind"] = kind
        intents[i]["sel_row"] = sel_row
        intents[i]["src_node"] = src_node
        intents[i]["dst_node"] = dst_node
        intents[i]["trace_begin"] = len(trs)
        trs.extend(tl)
        intents[i]["trace_end"] = len(trs)
        intents[i]["allowed"] = allowed
        expect[i] = (dsw, dport, -1)
    traces = np.zeros(max(len(trs), 1), TRACE_DT_LOCAL)
    for t, rec in enumerate(trs):
        traces[t] = rec
    return intents, expect, traces


TRACE_DT_LOCAL = np.dtype([("jmask", "<u4"), ("last_switch", "<i4"), ("last_port", "<u2"),
                           ("hops", "u1"), ("state", "u1")])


@pytest.mark.parametrize("case", _NET_CASES, ids=[c[0] for c in _NET_CASES])
def test_network_verdict_case(orc, case):
    """One hand-written network intent per case, judged alone."""
    intents, expect, traces = _net_case_arrays([case])
    pss, reason, summ, err = orc.report(intents, np.zeros((0, 1), np.uint64), np.zeros(0, np.uint32), 0,
                                        traces, expect, np.zeros(0, np.int32))
    assert err == 0
    assert reason[0] == case[-1], case[0]
    assert int(pss[0]) == (1 if case[-1] == 0 else 0)
    assert summ["counts"][2][case[-1]] == 1 and summ["counts"].sum() == 1


def test_network_verdict_cases_together(orc):
    """The same cases as one batch: reasons do not depend on neighbours."""
    intents, expect, traces = _net_case_arrays(_NET_CASES)
    pss, reason, summ, err = orc.report(intents, np.zeros((0, 1), np.uint64), np.zeros(0, np.uint32), 0,
                                        traces, expect, np.zeros(0, np.int32))
    assert err == 0
    assert list(reason) == [c[-1] for c in _NET_CASES]


def _one_row(nodes, N):
    W = (N + 63) // 64
    row = np.zeros((1, W), np.uint64)
    for n in nodes:
        row[0, n >> 6] |= np.uint64(1) << np.uint64(n & 63)
    return row, np.array([len(nodes)], np.uint32)


@pytest.mark.parametrize("row_nodes,src,dst,net_ok,expected", [
    ([], 3, 70, True, 1),            # empty row: NO_FEASIBLE_NODE, not ENDPOINT_INFEASIBLE
    ([], 3, 70, False, 1),           # ... and the compute code wins over a leak
    ([5], 3, 70, True, 2),           # non-empty row, neither endpoint admitted
    ([3], 3, 70, True, 2),           # only the source admitted
    ([70], 3, 70, True, 2),          # only the destination admitted
    ([3, 70], 3, 70, False, 4),      # endpoints fine, the trace leaks
    ([3, 70], 3, 70, True, 0),
    ([64], 64, 64, True, 0),         # same node at both ends, first bit of the second word
    ([63], 63, 64, True, 2),         # neighbouring bits across a word boundary
])
def test_hybrid_verdict_case(orc, row_nodes, src, dst, net_ok, expected):
    N = 100
    feas, pc = _one_row(row_nodes, N)
    tr = (0b01, 5, 2, 3, E) if net_ok else (0b11, 5, 2, 3, E)
    case = ("hybrid", 0b01, 5, 2, [tr], expected)
    intents, expect, traces = _net_case_arrays([case], kind=synth.KIND_HYBRID, sel_row=0, src_node=src,
                                               dst_node=dst)
    pss, reason, summ, err = orc.report(intents, feas, pc, N, traces, expect, np.zeros(0, np.int32))
    assert err == 0 and reason[0] == expected
    assert summ["counts"][3][expected] == 1


def test_compute_verdict_case(orc):
    """Compute-only intents read only the row's popcount."""
    N = 70
    feas = np.zeros((2, 2), np.uint64)
    feas[1, 1] = 1 << 3
    pc = np.array([0, 1], np.uint32)
    intents = np.zeros(2, synth.INTENT_DT)
    intents["kind"] = synth.KIND_COMPUTE
    intents["sel_row"] = [0, 1]
    expect = np.zeros(2, synth.EXPECT_DT)
    expect["reach_q"] = -1
    pss, reason, summ, err = orc.report(intents, feas, pc, N, np.zeros(1, TRACE_DT_LOCAL), expect,
                                        np.zeros(0, np.int32))
    assert list(reason) == [1, 0] and int(pss[0]) == 0b10
