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
from helpers import exact_rule, load_golden, ports_topology, tables_from_lists

REASONS = {"PASS": 0, "NO_FEASIBLE_NODE": 1, "ENDPOINT_INFEASIBLE": 2, "NO_FLOW": 3, "LEAK": 4,
           "UNDELIVERED": 5, "WRONG_EGRESS": 6, "MALFORMED": 7}


def _leak_fixture():
    fx = load_golden("paper_transit_leak.json")
    names = [s["name"] for s in fx["switches"]]
    nbr = [[names.index(x) for x in s["links"]] for s in fx["switches"]]
    jur = [fx["regions"].index(s["region"]) for s in fx["switches"]]
    topo = ports_topology(nbr, jur, hosts_per_switch=1)
    path = [names.index(x) for x in fx["flow"]["path"]]
    key = np.array([0x0A000001, 0x0A000003, (4000 << 16) | 443, 6], np.uint32)
    per = [[] for _ in names]
    for i, s in enumerate(path):
        a = topo["nbr"][s].index(path[i + 1]) if i + 1 < len(path) else len(topo["nbr"][s])
        per[s].append(exact_rule(key, a))
    rule_off, rules = tables_from_lists(per)
    return fx, topo, path, key, rule_off, rules


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
