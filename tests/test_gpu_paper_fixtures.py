"""The paper's own cases through the HIP path, against both the values the
fixtures state and the oracle:

- the 5-worker label matrix (Experimental Setup) with the label-schema
  selectors and the hallucinated-identifier failure mode, as selector rows;
- the transit switch of another region (failure mode 'Partial topology
  awareness': LEAK, and no compliant path exists) and the no-op network
  policy (failure mode 'Ambiguous path specification': NO_FLOW), traced,
  searched and judged on the GPU;
- a hallucinated label value failing closed (NO_FEASIBLE_NODE) and a
  hybrid endpoint placed on an infeasible node (ENDPOINT_INFEASIBLE)."""
import numpy as np
import pytest

import synth
from helpers import encode_label_matrix, encode_selector, leak_fixture, load_golden

pytestmark = pytest.mark.gpu

REASONS = {"PASS": 0, "NO_FEASIBLE_NODE": 1, "ENDPOINT_INFEASIBLE": 2, "NO_FLOW": 3, "LEAK": 4,
           "UNDELIVERED": 5, "WRONG_EGRESS": 6, "MALFORMED": 7}


@pytest.fixture(scope="module")
def g():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import gpu_run
    return gpu_run


def _label_rows():
    fx = load_golden("paper_label_matrix.json")
    labels, vocab = encode_label_matrix(fx)
    rows = [encode_selector(fx, vocab, c["selector"]) for c in fx["cases"]]
    off = np.zeros(len(rows) + 1, np.int32)
    off[1:] = np.cumsum([r.shape[0] for r in rows])
    preds = np.concatenate(rows) if rows else np.zeros(0, synth.PRED_DT)
    return fx, labels, off, preds


def test_paper_label_matrix_on_gpu(g, orc):
    fx, labels, off, preds = _label_rows()
    fg, pg = g.selectors(labels, off, preds)
    fo, po, err = orc.selectors(labels, off, preds)
    assert err == 0
    assert np.array_equal(fg, fo) and np.array_equal(pg, po)
    names = [n["name"] for n in fx["nodes"]]
    for i, c in enumerate(fx["cases"]):
        got = {names[n] for n in range(len(names)) if (int(fg[i, 0]) >> n) & 1}
        assert got == set(c["expect"]), c["cite"]
        assert pg[i] == len(c["expect"])


def test_paper_transit_leak_and_noop_on_gpu(g, orc):
    fx, topo, path, key, rule_off, rules = leak_fixture()
    S = topo["S"]
    hdr = key[None, :].copy()
    ing = np.array([path[0]], np.int32)
    tg = g.trace(S, topo["port_off"], topo["port_peer"], topo["jur"], rule_off, rules, hdr, ing, 16)
    to, err = orc.trace(S, topo["port_off"], topo["port_peer"], topo["jur"], rule_off, rules, hdr, ing, 16)
    assert err == 0
    for f in ("jmask", "last_switch", "last_port", "hops", "state"):
        assert np.array_equal(tg[f], to[f]), f
    assert tg[0]["state"] == 0 and tg[0]["hops"] == 2 and tg[0]["last_switch"] == path[-1]
    assert int(tg[0]["jmask"]) == 0b11          # both regions: the transit switch is in region-b
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
    src = np.full(I, path[0], np.int32)
    tgt = np.full(I, path[-1], np.int32)
    rg = g.reach(S, topo["adj_off"], topo["adj"], topo["jur"], src, allowed, tgt)
    ro, err = orc.reach(S, topo["adj_off"], topo["adj"], topo["jur"], src, allowed, tgt)
    assert err == 0 and np.array_equal(rg, ro)
    feas = np.zeros((1, 1), np.uint64)
    pc0 = np.zeros(1, np.uint32)
    pss, reason, summ = g.report(intents, feas, pc0, 0, tg, expect, rg)
    pso, reo, summo, err = orc.report(intents, feas, pc0, 0, to, expect, ro)
    assert err == 0
    assert np.array_equal(reason, reo) and np.array_equal(pss, pso)
    assert np.array_equal(summ["counts"], summo["counts"]) and np.array_equal(summ["no_path"], summo["no_path"])
    for i, c in enumerate(cases):
        assert reason[i] & 0x7F == REASONS[c["expect_reason"]], c["cite"]
        if "expect_no_path" in c:
            assert bool(reason[i] & 0x80) == c["expect_no_path"], c["cite"]
        if "expect_reach" in c:
            assert rg[i] == c["expect_reach"]
    assert reason[2] == REASONS["NO_FLOW"]       # the no-op policy reaches the GPU verdict


def test_paper_hallucinated_label_fails_closed_on_gpu(g, orc):
    fx = load_golden("paper_label_matrix.json")
    labels, vocab = encode_label_matrix(fx)
    p1 = encode_selector(fx, vocab, [["region", "In", ["eu_region"]]])
    p2 = encode_selector(fx, vocab, [["security", "In", ["high"]], ["zone", "In", ["cloud"]]])
    preds = np.concatenate([p1, p2])
    off = np.array([0, 1, 3], np.int32)
    fg, pg = g.selectors(labels, off, preds)
    intents = np.zeros(4, synth.INTENT_DT)
    intents["kind"] = [synth.KIND_COMPUTE, synth.KIND_COMPUTE, synth.KIND_HYBRID, synth.KIND_HYBRID]
    intents["sel_row"] = [0, 1, 1, 0]
    intents["src_node"] = [-1, -1, 3, 3]     # worker-4 (feasible for row 1) ...
    intents["dst_node"] = [-1, -1, 0, 3]     # ... worker-1 (edge zone: infeasible)
    intents["trace_begin"] = 0
    intents["trace_end"] = [0, 0, 1, 1]
    intents["allowed"] = 1
    expect = np.zeros(4, synth.EXPECT_DT)
    expect["dst_switch"] = -1
    expect["dst_port"] = -1
    expect["reach_q"] = -1
    tr = np.zeros(1, orc.TRACE_DT)
    tr[0] = (1, 0, 0, 0, 0)                  # a delivered, compliant trace: only placement can fail
    pss, reason, summ = g.report(intents, fg, pg, labels.shape[0], tr, expect, np.zeros(1, np.int32))
    pso, reo, _, err = orc.report(intents, fg, pg, labels.shape[0], tr, expect, np.zeros(1, np.int32))
    assert err == 0 and np.array_equal(reason, reo) and np.array_equal(pss, pso)
    assert list(reason) == [1, 0, 2, 1]      # the empty row reports NO_FEASIBLE_NODE before its endpoints
    assert int(pss[0]) == 0b0010
