"""Parity at the benchmark's full sizes, in the launch configuration the
benchmark times: the GPU computes every output and the oracle recomputes
every output (all cores), compared element by element; properties that
hold at any size are checked on top."""
import sys
import time

import numpy as np
import pytest

import synth

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]


def _say(*a):
    print("[fullsize]", *a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def g():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import gpu_run
    return gpu_run


def _popcount_rows(f):
    return np.unpackbits(f.view(np.uint8), axis=1).sum(1)


def _same(a, b, what):
    a, b = np.asarray(a), np.asarray(b)
    assert a.shape == b.shape, (what, a.shape, b.shape)
    if not np.array_equal(a, b):
        bad = np.argwhere(a != b)
        raise AssertionError(f"{what}: {bad.shape[0]} mismatches, first at {tuple(bad[0])}: "
                             f"gpu {a[tuple(bad[0])]} oracle {b[tuple(bad[0])]}")


def _same_traces(a, b):
    assert a.shape == b.shape
    for f in ("jmask", "last_switch", "last_port", "hops", "state"):
        _same(a[f], b[f], f"trace field {f}")


def test_cfg2_selectors_full(g, orc):
    t0 = time.time()
    wl = synth.cfg2()
    fg, pg = g.selectors(wl["labels"], wl["pred_off"], wl["preds"])
    N = wl["N"]
    W = (N + 63) // 64
    assert fg.shape == (wl["I_rows"], W)
    assert np.array_equal(_popcount_rows(fg), pg)                 # popcount is the row's bit count
    assert not np.any(fg[:, -1] >> np.uint64(N % 64))              # padding bits are zero
    _say(f"cfg2 gpu done {time.time() - t0:.1f} s")
    fo, po, err = orc.selectors(wl["labels"], wl["pred_off"], wl["preds"])
    _say(f"cfg2 oracle done {time.time() - t0:.1f} s")
    assert err == 0
    _same(fg, fo, "feasible")
    _same(pg, po, "popcnt")


def test_cfg3_trace_full(g, orc):
    t0 = time.time()
    wl = synth.cfg3()
    tg = g.trace(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"], wl["rules"], wl["hdr"],
                 wl["ingress"], wl["ttl"])
    _say(f"cfg3 gpu done {time.time() - t0:.1f} s")
    assert np.all(tg["state"] <= 3) and np.all(tg["hops"] <= wl["ttl"])
    eg = tg["state"] == 0
    assert np.all(tg["last_port"][~eg] == 0xFFFF)
    p = wl["port_off"][tg["last_switch"][eg]] + tg["last_port"][eg]
    assert np.all(wl["port_peer"][p] == -1)                          # egress only through host ports
    assert np.all((tg["jmask"] >> wl["jur"][wl["ingress"]].astype(np.uint32)) & 1)
    assert 0.5 < eg.mean() < 0.9
    to, err = orc.trace(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"], wl["rules"],
                        wl["hdr"], wl["ingress"], wl["ttl"])
    _say(f"cfg3 oracle done {time.time() - t0:.1f} s")
    assert err == 0
    _same_traces(tg, to)


def test_cfg4_reach_full(g, orc):
    t0 = time.time()
    wl = synth.cfg4()
    dg = g.reach(wl["V"], wl["adj_off"], wl["adj"], wl["region"], wl["src"], wl["allowed"])
    _say(f"cfg4 gpu done {time.time() - t0:.1f} s")
    assert dg.shape == (256, wl["V"])
    assert np.all(dg[np.arange(256), wl["src"]] == 0)
    do, err = orc.reach(wl["V"], wl["adj_off"], wl["adj"], wl["region"], wl["src"], wl["allowed"])
    _say(f"cfg4 oracle done {time.time() - t0:.1f} s")
    assert err == 0
    _same(dg, do, "dist")
    # every reached vertex is allowed and has a parent one layer up (sampled rows)
    adj_off, adj, region = wl["adj_off"], wl["adj"], wl["region"]
    src = np.repeat(np.arange(wl["V"]), np.diff(adj_off))
    for q in range(0, 256, 16):
        d = dg[q]
        A = int(wl["allowed"][q])
        reached = d >= 0
        assert np.all((A >> region[reached].astype(np.int64)) & 1)
        ok_e = reached[src] & reached[adj]
        assert np.all(np.abs(d[src[ok_e]] - d[adj[ok_e]]) <= 1)


def test_cfg5_end_to_end_full(g, orc):
    t0 = time.time()
    wl = synth.cfg5()
    _say(f"cfg5 generated {time.time() - t0:.1f} s")
    gp = g.run_workload(wl)
    _say(f"cfg5 gpu done {time.time() - t0:.1f} s")
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
    # the oracle on the whole job
    oo = orc.run_workload(wl)
    _say(f"cfg5 oracle done {time.time() - t0:.1f} s")
    _same(gp["feasible"], oo["feasible"], "feasible")
    _same(gp["popcnt"], oo["popcnt"], "popcnt")
    _same_traces(gp["traces"], oo["traces"])
    _same(gp["reach"], oo["reach"], "reach")
    _same(gp["reason"], oo["reason"], "reason")
    _same(gp["pass"], oo["pass"], "pass")
    for f in ("counts", "no_path"):
        _same(gp["summary"][f], oo["summary"][f], f"summary {f}")
    flags = oo["sel_err"] | oo["trace_err"] | oo["reach_err"] | oo["report_err"]
    assert gp["flags"] == flags == 0
