"""Pins of the oracle's visited-switch summaries and of the locality that
incremental re-validation after rule changes relies on.

- The summary (bit s mod 64 of every switch on the walk) against the test
  suite's own brute-force walker, on a dense small graph (every terminal
  state, loops) and on a fat-tree of 80 switches (bits shared mod 64).
- Locality: after rewriting the rules of a few switches, every walk whose
  old summary has no bit of a changed switch is the same walk (same record,
  same summary) on the new tables, while some walks do change.
"""
import numpy as np
import pytest

import synth
from test_oracle_trace import _first_match


def _walk_path(S, port_off, port_peer, rule_off, rules, h, s, ttl):
    """The switches a brute-force walk visits (ingress first)."""
    path, hops = [s], 0
    while True:
        r = _first_match(rules, int(rule_off[s]), int(rule_off[s + 1]), h)
        if r < 0:
            return path
        a = int(rules[r]["action"])
        if a == 0xFFFF:
            return path
        peer = int(port_peer[port_off[s] + a])
        if peer == -1 or hops == ttl:
            return path
        s, hops = peer, hops + 1
        path.append(s)


def _workloads():
    return [("cfg1-dense", synth.cfg1(0, "dense")),
            ("fat-tree-80", synth.trace_workload(5, 8, 4, 24, 300, 12, 200, variant="dense"))]


@pytest.mark.parametrize("name,wl", _workloads())
def test_summary_matches_walker(orc, name, wl):
    out, vsum, walk, err = orc.trace(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"],
                                     wl["rules"], wl["hdr"], wl["ingress"], wl["ttl"], summary=True)
    assert err == 0
    long_walks = 0
    for t in range(wl["hdr"].shape[0]):
        path = _walk_path(wl["S"], wl["port_off"], wl["port_peer"], wl["rule_off"], wl["rules"], wl["hdr"][t],
                          int(wl["ingress"][t]), wl["ttl"])
        want = 0
        for s in path:
            want |= 1 << (s & 63)
        assert int(vsum[t]) == want, (name, t, path)
        rec = (path + [-1] * 8)[:8]
        assert walk[t].tolist() == rec, (name, t, path)
        assert int(out[t]["hops"]) + 1 == len(path)
        long_walks += len(path) > 8
    assert long_walks > 0  # walks past 8 switches keep their first 8
    if wl["S"] > 64:
        assert any(int(v) >> 16 & 1 for v in vsum)  # switch 16 and 80 share a bit, and walks get there


def test_invalid_ingress_has_empty_summary(orc):
    wl = synth.cfg1(0, "rpath")
    ingress = wl["ingress"].copy()
    ingress[:3] = [-1, wl["S"], 10 ** 6]
    out, vsum, walk, err = orc.trace(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"],
                                     wl["rules"], wl["hdr"], ingress, wl["ttl"], summary=True)
    assert (vsum[:3] == 0).all() and (vsum[3:] != 0).all()
    assert (walk[:3] == -1).all() and (walk[3:, 0] == ingress[3:]).all()


@pytest.mark.parametrize("resize", [False, True])
@pytest.mark.parametrize("name,wl", _workloads())
def test_walks_that_miss_the_changed_switches_are_unchanged(orc, name, wl, resize):
    S = wl["S"]
    rng = np.random.default_rng(7)
    changed = rng.choice(S, size=3, replace=False)
    r_off2, rules2 = synth.mutate_tables(7, wl["port_off"], wl["rule_off"], wl["rules"], changed, resize=resize)
    args = (S, wl["port_off"], wl["port_peer"], wl["jur"])
    o1, v1, w1, _ = orc.trace(*args, wl["rule_off"], wl["rules"], wl["hdr"], wl["ingress"], wl["ttl"], summary=True)
    o2, v2, w2, _ = orc.trace(*args, r_off2, rules2, wl["hdr"], wl["ingress"], wl["ttl"], summary=True)
    cmask = 0
    for s in changed:
        cmask |= 1 << (int(s) & 63)
    marked = (v1 & np.uint64(cmask)) != 0
    keep = ~marked
    assert np.array_equal(o1[keep], o2[keep]) and np.array_equal(v1[keep], v2[keep])
    assert np.array_equal(w1[keep], w2[keep])
    assert marked.sum() > 0 and (o1[marked] != o2[marked]).any()
    # exact for walks of at most 8 switches (their record lists them all), the
    # summary for longer ones: every walk this keeps is unchanged too
    short = o1["hops"].astype(np.int64) + 1 <= 8
    hit = np.isin(w1, changed).any(axis=1)
    keep2 = np.where(short, ~hit, keep)
    assert np.array_equal(o1[keep2], o2[keep2]) and np.array_equal(v1[keep2], v2[keep2])
    assert np.array_equal(w1[keep2], w2[keep2])
    assert keep2.sum() >= keep.sum()
    if wl["S"] > 64:  # bits are shared: the walk records keep walks the summary would re-trace
        assert (keep2 & ~keep).sum() > 0
