"""Pins for the oracle's flow trace (routing constraints on realised paths).

Pins: a per-bit, sort-then-scan brute force of first match; exact-match
rules compiled along shortest paths (the trace reduces to BFS); masked
shortest paths (reduces to masked BFS); a two-switch ping-pong loop whose
TTL outcome has a closed form; the literal i.i.d. reading's closed form
(every lookup misses); invariants on every terminal record.
"""
import networkx as nx
import numpy as np
import pytest

import synth
from helpers import exact_rule, line_topology, ports_topology, tables_from_lists


def _bit_match(rule, h):
    for w in range(4):
        for b in range(32):
            if (int(rule["mask"][w]) >> b) & 1 and ((int(rule["value"][w]) >> b) & 1) != ((int(h[w]) >> b) & 1):
                return False
    return True


def _first_match(rules, lo, hi, h):
    """Sort the switch's rules by (priority desc, index asc) and take the first match."""
    order = sorted(range(lo, hi), key=lambda r: (-int(rules[r]["priority"]), r))
    for r in order:
        if _bit_match(rules[r], h):
            return r
    return -1


def _walk(S, port_off, port_peer, jur, rule_off, rules, h, s, ttl):
    """Brute-force walker built on _first_match."""
    jm, hops = 1 << int(jur[s]), 0
    while True:
        r = _first_match(rules, int(rule_off[s]), int(rule_off[s + 1]), h)
        if r < 0:
            return jm, s, 0xFFFF, hops, 2
        a = int(rules[r]["action"])
        if a == 0xFFFF:
            return jm, s, 0xFFFF, hops, 1
        peer = int(port_peer[port_off[s] + a])
        if peer == -1:
            return jm, s, a, hops, 0
        if hops == ttl:
            return jm, s, 0xFFFF, hops, 3
        s, hops = peer, hops + 1
        jm |= 1 << int(jur[s])


def _check_against_walker(orc, wl, ttl=None):
    ttl = wl["ttl"] if ttl is None else ttl
    out, err = orc.trace(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"],
                         wl["rules"], wl["hdr"], wl["ingress"], ttl)
    assert err == 0
    for t in range(wl["hdr"].shape[0]):
        want = _walk(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"], wl["rules"],
                     wl["hdr"][t], int(wl["ingress"][t]), ttl)
        got = tuple(int(out[t][f]) for f in ("jmask", "last_switch", "last_port", "hops", "state"))
        assert got == want, t
    return out


@pytest.mark.parametrize("variant", ["rpath", "dense"])
def test_walker_cfg1(orc, variant):
    wl = synth.cfg1(0, variant)
    out = _check_against_walker(orc, wl)
    if variant == "dense":
        # the dense reading must exercise every terminal state and TTL
        assert set(np.unique(out["state"])) == {0, 1, 2, 3}


def test_walker_small_dense_ties(orc):
    """Priorities in [0, 8) make equal-priority matches common: the lower
    index must win."""
    rng = np.random.default_rng(3)
    topo = synth.random_graph(rng, 7, 10, 2, 4)
    rule_off, rules, _ = synth.build_tables(rng, topo, 24, 0.03, prio="small", prio_range=3)
    T = 400
    hdr = synth.random_keys(rng, T)
    ingress = rng.integers(0, 7, size=T).astype(np.int32)
    wl = synth.Workload("t", 3)
    wl.arrays.update(port_off=topo["port_off"], port_peer=topo["port_peer"], jur=topo["jur"],
                     rule_off=rule_off, rules=rules, hdr=hdr, ingress=ingress)
    wl.sizes.update(S=7, ttl=9)
    out = _check_against_walker(orc, wl)
    # ties really happened: some lookups had several matches at the top priority
    ties = 0
    for t in range(T):
        s = int(ingress[t])
        lo, hi = int(rule_off[s]), int(rule_off[s + 1])
        m = [r for r in range(lo, hi) if _bit_match(rules[r], hdr[t])]
        if len(m) > 1:
            top = max(int(rules[r]["priority"]) for r in m)
            ties += sum(int(rules[r]["priority"]) == top for r in m) > 1
    assert ties > 10


def test_exact_rules_along_shortest_paths(orc):
    """Exact-match rules compiled along a BFS shortest path: every trace
    egresses at the destination host after exactly dist(src, dst) links."""
    rng = np.random.default_rng(8)
    topo = synth.random_graph(rng, 15, 24, 1, 3)
    G = nx.Graph()
    G.add_nodes_from(range(15))
    for s in range(15):
        for v in topo["nbr"][s]:
            G.add_edge(s, v)
    per = [[] for _ in range(15)]
    hdr, ingress, want = [], [], []
    for f in range(60):
        u, v = (int(x) for x in rng.choice(15, size=2, replace=False))
        path = nx.shortest_path(G, u, v)
        key = np.array([f, 7 * f + 1, (f << 16) | 80, 6], np.uint32)
        for i, s in enumerate(path):
            a = topo["nbr"][s].index(path[i + 1]) if i + 1 < len(path) else len(topo["nbr"][s])
            per[s].append(exact_rule(key, a))
        hdr.append(key)
        ingress.append(u)
        want.append((v, len(path) - 1))
    rule_off, rules = tables_from_lists(per)
    out, err = orc.trace(15, topo["port_off"], topo["port_peer"], topo["jur"], rule_off, rules,
                         np.array(hdr), np.array(ingress, np.int32), 32)
    assert err == 0
    for t, (v, d) in enumerate(want):
        assert out[t]["state"] == orc.EGRESS and out[t]["last_switch"] == v and out[t]["hops"] == d


def test_masked_paths_are_compliant(orc):
    """Rules compiled along shortest paths of the allowed-induced subgraph:
    the trace is compliant (jmask within allowed) and hops = masked distance."""
    rng = np.random.default_rng(21)
    S = 30
    topo = synth.random_graph(rng, S, 50, 1, 4)
    jur = topo["jur"]
    per = [[] for _ in range(S)]
    hdr, ingress, checks = [], [], []
    for f in range(80):
        allowed = int(rng.integers(1, 16))
        ok = [s for s in range(S) if (allowed >> int(jur[s])) & 1]
        G = nx.Graph()
        G.add_nodes_from(ok)
        G.add_edges_from((s, v) for s in ok for v in topo["nbr"][s] if v in ok)
        if len(ok) < 2:
            continue
        u, v = (int(x) for x in rng.choice(ok, size=2, replace=False))
        if not nx.has_path(G, u, v):
            continue
        path = nx.shortest_path(G, u, v)
        key = np.array([f, f + 3, f * 11, 17], np.uint32)
        for i, s in enumerate(path):
            a = topo["nbr"][s].index(path[i + 1]) if i + 1 < len(path) else len(topo["nbr"][s])
            per[s].append(exact_rule(key, a))
        hdr.append(key)
        ingress.append(u)
        checks.append((allowed, v, len(path) - 1))
    rule_off, rules = tables_from_lists(per)
    out, err = orc.trace(S, topo["port_off"], topo["port_peer"], jur, rule_off, rules,
                         np.array(hdr), np.array(ingress, np.int32), 32)
    assert len(checks) > 20
    for t, (allowed, v, d) in enumerate(checks):
        assert int(out[t]["jmask"]) & ~allowed == 0
        assert out[t]["state"] == orc.EGRESS and out[t]["last_switch"] == v and out[t]["hops"] == d


@pytest.mark.parametrize("ttl", [0, 1, 2, 5, 16, 255])
def test_ping_pong_ttl(orc, ttl):
    """Two switches forwarding the header to each other: TTL after exactly
    `ttl` links, ending at the ingress iff ttl is even."""
    topo = line_topology(2, [0, 1])
    key = np.array([1, 2, 3, 4], np.uint32)
    rule_off, rules = tables_from_lists([[exact_rule(key, 0)], [exact_rule(key, 0)]])
    out, err = orc.trace(2, topo["port_off"], topo["port_peer"], topo["jur"], rule_off, rules,
                         key[None, :], np.array([0], np.int32), ttl)
    r = out[0]
    assert r["state"] == orc.TTL and r["hops"] == ttl
    assert r["last_switch"] == (0 if ttl % 2 == 0 else 1)
    assert r["jmask"] == (1 if ttl == 0 else 3)


def test_literal_reading_misses_at_ingress(orc):
    """Literal i.i.d. rules (50% wildcards over 104 bits) match a uniform
    header with probability 0.75^104 ~ 1e-13 per rule: every trace misses
    at its ingress with zero hops."""
    wl = synth.cfg1(0, "literal")
    out, err = orc.trace(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"],
                         wl["rules"], wl["hdr"], wl["ingress"], wl["ttl"])
    assert np.all(out["state"] == orc.MISS) and np.all(out["hops"] == 0)
    assert np.array_equal(out["last_switch"], wl["ingress"])
    assert np.array_equal(out["jmask"], (1 << wl["jur"][wl["ingress"]].astype(np.uint32)))


def _graph(wl):
    G = nx.Graph()
    G.add_nodes_from(range(wl["S"]))
    for s in range(wl["S"]):
        for p in range(wl["port_off"][s], wl["port_off"][s + 1]):
            if wl["port_peer"][p] >= 0:
                G.add_edge(s, int(wl["port_peer"][p]))
    return G


@pytest.mark.parametrize("variant", ["rpath", "dense", "literal"])
def test_terminal_invariants(orc, variant):
    wl = synth.trace_workload(4, 8, 4, 128, 3000, 12, 800, variant=variant)
    out, err = orc.trace(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"],
                         wl["rules"], wl["hdr"], wl["ingress"], wl["ttl"])
    assert err == 0
    G = _graph(wl)
    dist = dict(nx.all_pairs_shortest_path_length(G))
    for t in range(out.shape[0]):
        r = out[t]
        s0, s1 = int(wl["ingress"][t]), int(r["last_switch"])
        assert r["state"] in (0, 1, 2, 3)
        assert r["hops"] <= wl["ttl"]
        jm = int(r["jmask"])
        assert (jm >> int(wl["jur"][s0])) & 1 and (jm >> int(wl["jur"][s1])) & 1
        assert dist[s0][s1] <= r["hops"]
        if r["state"] == orc.EGRESS:
            p = int(wl["port_off"][s1]) + int(r["last_port"])
            assert wl["port_peer"][p] == -1
        else:
            assert r["last_port"] == 0xFFFF
        if r["state"] == orc.TTL:
            assert r["hops"] == wl["ttl"]


def test_rpath_delivers_most_flows(orc):
    """R-path tables: a header follows its compiled path unless a rule on it
    drops (5%) or mis-routes (2%); with 5 switches on most paths about
    (0.93)^5 ~ 70% egress."""
    wl = synth.trace_workload(4, 8, 4, 256, 4000, 32, 1000)
    out, _ = orc.trace(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"],
                       wl["rules"], wl["hdr"], wl["ingress"], wl["ttl"])
    frac = np.mean(out["state"] == orc.EGRESS)
    assert 0.55 < frac < 0.85


def test_malformed_inputs(orc):
    topo = line_topology(3, [0, 1, 40])
    key = np.array([1, 2, 3, 4], np.uint32)
    per = [[exact_rule(key, 0)], [exact_rule(key, 1)], [exact_rule(key, 9)]]
    rule_off, rules = tables_from_lists(per)
    hdr = np.stack([key] * 4)
    ingress = np.array([0, 7, -1, 2], np.int32)
    out, err = orc.trace(3, topo["port_off"], topo["port_peer"], topo["jur"], rule_off, rules, hdr, ingress, 8)
    assert err & orc.F_SWITCH and err & orc.F_JUR and err & orc.F_ACTION
    # trace 0: 0 -> 1 -> 2, whose jurisdiction 40 is out of range; action 9 > ports
    assert out[0]["state"] == orc.MISS and out[0]["last_switch"] == 2 and out[0]["hops"] == 2
    assert out[0]["jmask"] == 0b11
    for t in (1, 2):
        assert out[t]["state"] == orc.MISS and out[t]["jmask"] == 0 and out[t]["hops"] == 0
    bad_off = rule_off.copy()
    bad_off[1] = 99
    out, err = orc.trace(3, topo["port_off"], topo["port_peer"], topo["jur"], bad_off, rules, hdr[:1],
                         ingress[:1], 8)
    assert err & orc.F_OFFSETS and out[0]["state"] == orc.MISS


def test_switch_without_rules_misses(orc):
    topo = ports_topology([[1], [0]], [0, 1])
    rule_off = np.zeros(3, np.int32)
    rules = np.zeros(0, synth.RULE_DT)
    out, err = orc.trace(2, topo["port_off"], topo["port_peer"], topo["jur"], rule_off, rules,
                         np.zeros((1, 4), np.uint32), np.array([1], np.int32), 4)
    assert out[0]["state"] == orc.MISS and out[0]["hops"] == 0 and out[0]["last_switch"] == 1
