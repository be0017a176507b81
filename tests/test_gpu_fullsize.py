"""Parity at the benchmark's full sizes, in the launch configuration the
benchmark times: the GPU computes every output, the oracle recomputes a
seeded sample of them one by one, and properties that hold at any size are
checked on every output."""
import numpy as np
import pytest

import synth

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]


@pytest.fixture(scope="module")
def g():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import gpu_run
    return gpu_run


def _popcount_rows(f):
    return np.unpackbits(f.view(np.uint8), axis=1).sum(1)


def test_cfg2_selectors_full(g, orc):
    wl = synth.cfg2()
    fg, pg = g.selectors(wl["labels"], wl["pred_off"], wl["preds"])
    N = wl["N"]
    W = (N + 63) // 64
    assert fg.shape == (wl["I_rows"], W)
    assert np.array_equal(_popcount_rows(fg), pg)                 # popcount is the row's bit count
    assert not np.any(fg[:, -1] >> np.uint64(N % 64))              # padding bits are zero
    rows = np.unique(np.r_[0, wl["I_rows"] - 1, np.random.default_rng(0).integers(0, wl["I_rows"], 62)]).astype(np.int32)
    fo, po, err = orc.selectors(wl["labels"], wl["pred_off"], wl["preds"], rows=rows)
    assert np.array_equal(fg[rows], fo) and np.array_equal(pg[rows], po) and err == 0


def test_cfg3_trace_full(g, orc):
    wl = synth.cfg3()
    tg = g.trace(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"], wl["rules"], wl["hdr"],
                 wl["ingress"], wl["ttl"])
    assert np.all(tg["state"] <= 3) and np.all(tg["hops"] <= wl["ttl"])
    eg = tg["state"] == 0
    assert np.all(tg["last_port"][~eg] == 0xFFFF)
    p = wl["port_off"][tg["last_switch"][eg]] + tg["last_port"][eg]
    assert np.all(wl["port_peer"][p] == -1)                          # egress only through host ports
    assert np.all((tg["jmask"] >> wl["jur"][wl["ingress"]].astype(np.uint32)) & 1)
    idx = np.random.default_rng(1).choice(wl["T"], 3000, replace=False)
    to, err = orc.trace(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"], wl["rules"],
                        wl["hdr"], wl["ingress"], wl["ttl"], idx=idx)
    assert err == 0
    for f in ("jmask", "last_switch", "last_port", "hops", "state"):
        assert np.array_equal(tg[f][idx], to[f]), f
    assert 0.5 < eg.mean() < 0.9


def test_cfg4_reach_full(g, orc):
    wl = synth.cfg4()
    dg = g.reach(wl["V"], wl["adj_off"], wl["adj"], wl["region"], wl["src"], wl["allowed"])
    assert dg.shape == (256, wl["V"])
    assert np.all(dg[np.arange(256), wl["src"]] == 0)
    qs = np.random.default_rng(2).choice(256, 6, replace=False)
    do, err = orc.reach(wl["V"], wl["adj_off"], wl["adj"], wl["region"], wl["src"], wl["allowed"], qidx=qs)
    assert err == 0 and np.array_equal(dg[qs], do)
    # every reached vertex is allowed and has a parent one layer up (all rows)
    adj_off, adj, region = wl["adj_off"], wl["adj"], wl["region"]
    src = np.repeat(np.arange(wl["V"]), np.diff(adj_off))
    for q in range(0, 256, 16):
        d = dg[q]
        A = int(wl["allowed"][q])
        reached = d >= 0
        assert np.all((A >> region[reached].astype(np.int64)) & 1)
        ok_e = reached[src] & reached[adj]
        assert np.all(np.abs(d[src[ok_e]] - d[adj[ok_e]]) <= 1)


def test_cfg5_end_to_end_sampled(g, orc):
    import bench
    wl = synth.cfg5()
    gp = g.run_workload(wl)
    assert gp["flags"] == 0
    I = wl["I"]
    reason = gp["reason"]
    bits = np.unpackbits(gp["pass"].view(np.uint8), bitorder="little")[:I]
    assert np.array_equal(bits == 1, (reason & 0x7F) == 0)
    hist = np.zeros((4, 16), np.uint64)
    np.add.at(hist, (wl["intents"]["kind"] & 3, reason & 0x7F), 1)
    assert np.array_equal(gp["summary"]["counts"], hist)
    # a passing network intent has a compliant path no longer than its trace
    it, ex = wl["intents"], wl["expect"]
    net = np.flatnonzero(((it["kind"] & 2) != 0) & (bits == 1))
    d = gp["reach"][ex["reach_q"][net]]
    hops = gp["traces"]["hops"][it["trace_begin"][net]]
    assert np.all(d >= 0) and np.all(d <= hops)
    # oracle on every 512th intent, with the rows, traces and queries it uses
    sp = bench.sample_subproblem(wl, 512)
    feas, pc, _ = orc.selectors(wl["labels"], wl["pred_off"], wl["preds"], rows=sp["rows"])
    assert np.array_equal(feas, gp["feasible"][sp["rows"]]) and np.array_equal(pc, gp["popcnt"][sp["rows"]])
    tr, _ = orc.trace(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"], wl["rules"], wl["hdr"],
                      wl["ingress"], wl["ttl"], idx=sp["traces"])
    for f in ("jmask", "last_switch", "last_port", "hops", "state"):
        assert np.array_equal(tr[f], gp["traces"][f][sp["traces"]]), f
    rc, _ = orc.reach(wl["V"], wl["adj_off"], wl["adj"], wl["region"], wl["src"], wl["allowed"], wl["target"],
                      qidx=sp["queries"])
    assert np.array_equal(rc, gp["reach"][sp["queries"]])
    _, ro, _, _ = orc.report(sp["intents"], feas, pc, wl["N"], tr, sp["expect"], rc)
    assert np.array_equal(ro, reason[np.arange(0, I, 512)])
