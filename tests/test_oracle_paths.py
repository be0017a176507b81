"""Pins for the oracle's waypoint and forbidden-switch checks (the paper's
routing constraints: required waypoints and forbidden vertices, checked over
realised paths by the validator).

Pins: a sort-then-scan walker that records the visited switches; exact-match
rules along shortest paths (the visited set is the path); the two-switch
ping-pong loop; a layered-state breadth-first search over (vertex, waypoints
reached) that finds the shortest constrained walk without splitting it into
legs; networkx shortest paths per leg on the induced subgraph with the
forbidden switches removed; closed forms on a path, a cycle and a fat-tree;
hand-built verdict fixtures.
"""
from collections import deque

import networkx as nx
import numpy as np
import pytest

import synth
from helpers import exact_rule, line_topology, ports_topology, tables_from_lists


# ---------------------------------------------------------------- traces

def _first_match(rules, lo, hi, h):
    order = sorted(range(lo, hi), key=lambda r: (-int(rules[r]["priority"]), r))
    for r in order:
        ok = all(((int(h[w]) ^ int(rules[r]["value"][w])) & int(rules[r]["mask"][w])) == 0 for w in range(4))
        if ok:
            return r
    return -1


def _visited(wl, h, s, ttl):
    """Switches a header visits from ingress s (sort-based first match)."""
    seen = [s]
    hops = 0
    while True:
        r = _first_match(wl["rules"], int(wl["rule_off"][s]), int(wl["rule_off"][s + 1]), h)
        if r < 0:
            return seen
        a = int(wl["rules"][r]["action"])
        if a == 0xFFFF:
            return seen
        peer = int(wl["port_peer"][wl["port_off"][s] + a])
        if peer == -1 or hops == ttl:
            return seen
        s, hops = peer, hops + 1
        seen.append(s)


def _watch_trace(orc, wl, watch, ttl=None):
    ttl = wl["ttl"] if ttl is None else ttl
    return orc.trace(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"], wl["rules"], wl["hdr"],
                     wl["ingress"], ttl, watch=watch)


@pytest.mark.parametrize("variant", ["rpath", "dense"])
def test_visit_words_match_walker(orc, variant):
    wl = synth.cfg1(0, variant)
    rng = np.random.default_rng(11)
    T, S = wl["hdr"].shape[0], wl["S"]
    watch = rng.integers(-1, S, size=(T, 5)).astype(np.int32)
    watch[:, 0] = wl["ingress"]  # the ingress always counts as visited
    out, visit, err = _watch_trace(orc, wl, watch)
    assert err == 0
    plain, _ = orc.trace(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"], wl["rules"],
                         wl["hdr"], wl["ingress"], wl["ttl"])
    assert np.array_equal(out, plain)  # watching changes no trace record
    assert np.all(visit & 1)
    n_multi = 0
    for t in range(T):
        seen = set(_visited(wl, wl["hdr"][t], int(wl["ingress"][t]), wl["ttl"]))
        want = sum(1 << k for k in range(5) if int(watch[t, k]) in seen)
        assert int(visit[t]) == want, t
        n_multi += bin(want).count("1") > 2
    assert n_multi > 20


def test_visit_is_the_compiled_path(orc):
    """Exact rules along shortest paths: a trace visits exactly its path."""
    rng = np.random.default_rng(5)
    S = 16
    topo = synth.random_graph(rng, S, 26, 1, 3)
    G = nx.Graph()
    G.add_nodes_from(range(S))
    G.add_edges_from((s, v) for s in range(S) for v in topo["nbr"][s])
    per = [[] for _ in range(S)]
    hdr, ingress, paths = [], [], []
    for f in range(50):
        u, v = (int(x) for x in rng.choice(S, size=2, replace=False))
        path = nx.shortest_path(G, u, v)
        key = np.array([f, 3 * f + 2, (f << 16) | 443, 17], np.uint32)
        for i, s in enumerate(path):
            a = topo["nbr"][s].index(path[i + 1]) if i + 1 < len(path) else len(topo["nbr"][s])
            per[s].append(exact_rule(key, a))
        hdr.append(key)
        ingress.append(u)
        paths.append(set(path))
    rule_off, rules = tables_from_lists(per)
    watch = np.tile(np.arange(S, dtype=np.int32), (len(hdr), 1))  # slot k watches switch k
    out, visit, err = orc.trace(S, topo["port_off"], topo["port_peer"], topo["jur"], rule_off, rules,
                                np.array(hdr), np.array(ingress, np.int32), 32, watch=watch)
    assert err == 0
    for t, p in enumerate(paths):
        assert out[t]["state"] == orc.EGRESS
        assert int(visit[t]) == sum(1 << s for s in p)


@pytest.mark.parametrize("ttl", [0, 1, 2, 7])
def test_visit_ping_pong(orc, ttl):
    topo = line_topology(2, [0, 1])
    key = np.array([1, 2, 3, 4], np.uint32)
    rule_off, rules = tables_from_lists([[exact_rule(key, 0)], [exact_rule(key, 0)]])
    watch = np.array([[1, 0, -1]], np.int32)
    out, visit, err = orc.trace(2, topo["port_off"], topo["port_peer"], topo["jur"], rule_off, rules, key[None, :],
                                np.array([0], np.int32), ttl, watch=watch)
    assert out[0]["state"] == orc.TTL
    assert int(visit[0]) == (0b10 if ttl == 0 else 0b11)


def test_visit_malformed(orc):
    topo = line_topology(3, [0, 1, 2])
    key = np.array([1, 2, 3, 4], np.uint32)
    rule_off, rules = tables_from_lists([[exact_rule(key, 0)], [exact_rule(key, 1)], [exact_rule(key, 1)]])
    hdr = np.stack([key] * 2)
    watch = np.array([[2, 99, -5], [0, 1, 2]], np.int32)
    out, visit, err = orc.trace(3, topo["port_off"], topo["port_peer"], topo["jur"], rule_off, rules, hdr,
                                np.array([0, 9], np.int32), 8, watch=watch)
    assert err & orc.F_SWITCH
    assert out[0]["state"] == orc.EGRESS and int(visit[0]) == 0b001  # 0 -> 1 -> 2, host port of 2
    assert out[1]["state"] == orc.MISS and int(visit[1]) == 0  # ingress out of range


# ---------------------------------------------------------------- reach

def _usable(region, A, fb, v):
    return ((A >> int(region[v])) & 1) and v not in fb


def _layered(V, adj_off, adj, region, A, s, t, way, fb):
    """Shortest walk s -> way[0] -> ... -> t over usable vertices by BFS over
    states (vertex, number of waypoints reached in order)."""
    m = len(way)
    if not (0 <= s < V and 0 <= t < V) or not _usable(region, A, fb, s):
        return -1

    def advance(v, j):
        while j < m and way[j] == v:
            j += 1
        return j

    start = (s, advance(s, 0))
    dist = {start: 0}
    dq = deque([start])
    while dq:
        u, j = dq.popleft()
        if (u, j) == (t, m):
            return dist[(u, j)]
        for p in range(adj_off[u], adj_off[u + 1]):
            v = int(adj[p])
            if not _usable(region, A, fb, v):
                continue
            st = (v, advance(v, j))
            if st not in dist:
                dist[st] = dist[(u, j)] + 1
                dq.append(st)
    return -1


def _random_graph(rng, V, E, R):
    edges = set()
    while len(edges) < E:
        u, v = (int(x) for x in rng.integers(0, V, size=2))
        if u != v:
            edges.add((min(u, v), max(u, v)))
    nbr = [[] for _ in range(V)]
    for u, v in edges:
        nbr[u].append(v)
        nbr[v].append(u)
    adj_off = np.zeros(V + 1, np.int32)
    adj = []
    for u in range(V):
        adj.extend(sorted(nbr[u]))
        adj_off[u + 1] = len(adj)
    region = rng.integers(0, R, size=V).astype(np.uint8)
    return adj_off, np.asarray(adj, np.int32), region


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_via_layered_bfs(orc, seed):
    rng = np.random.default_rng(seed)
    V, Q, Kv, Kf = 24, 300, 3, 3
    adj_off, adj, region = _random_graph(rng, V, 40, 4)
    src = rng.integers(0, V, size=Q).astype(np.int32)
    target = rng.integers(0, V, size=Q).astype(np.int32)
    allowed = rng.integers(1, 16, size=Q).astype(np.uint32)
    via = rng.integers(0, V, size=(Q, Kv)).astype(np.int32)
    m = rng.integers(0, Kv + 1, size=Q)
    for q in range(Q):
        via[q, m[q]:] = -1
    via[::7, 1] = via[::7, 0]  # repeated waypoints
    forbid = rng.integers(-1, V, size=(Q, Kf)).astype(np.int32)
    forbid[::3] = -1
    dist, err = orc.reach_via(V, adj_off, adj, region, src, allowed, target, via, forbid)
    assert err == 0
    found = 0
    for q in range(Q):
        way = [int(x) for x in via[q, : m[q]]]
        fb = {int(x) for x in forbid[q] if x >= 0}
        want = _layered(V, adj_off, adj, region, int(allowed[q]), int(src[q]), int(target[q]), way, fb)
        assert int(dist[q]) == want, q
        found += want > 0
    assert found > 30


def test_via_networkx_legs(orc):
    wl = synth.rgg_workload(9, 1500, 6, 40, mean_degree=7.0, full_rows=False)
    rng = np.random.default_rng(9)
    V, Q = wl["V"], 40
    target = rng.integers(0, V, size=Q).astype(np.int32)
    via = rng.integers(0, V, size=(Q, 2)).astype(np.int32)
    forbid = rng.integers(0, V, size=(Q, 4)).astype(np.int32)
    dist, err = orc.reach_via(V, wl["adj_off"], wl["adj"], wl["region"], wl["src"], wl["allowed"], target, via,
                              forbid)
    assert err == 0
    for q in range(Q):
        A = int(wl["allowed"][q])
        fb = set(int(x) for x in forbid[q])
        ok = [v for v in range(V) if (A >> int(wl["region"][v])) & 1 and v not in fb]
        oks = set(ok)
        G = nx.Graph()
        G.add_nodes_from(ok)
        G.add_edges_from((u, int(wl["adj"][p])) for u in ok for p in range(wl["adj_off"][u], wl["adj_off"][u + 1])
                         if int(wl["adj"][p]) in oks)
        stops = [int(wl["src"][q])] + [int(x) for x in via[q]] + [int(target[q])]
        total = 0
        for a, b in zip(stops[:-1], stops[1:]):
            if a not in G or b not in G or not nx.has_path(G, a, b):
                total = -1
                break
            total += nx.shortest_path_length(G, a, b)
        assert int(dist[q]) == total, q


def test_via_closed_forms(orc):
    # path 0 - 1 - ... - 9, everything allowed
    n = 10
    topo = line_topology(n, [0] * n)
    region = np.zeros(n, np.uint8)
    src = np.array([2, 2, 2, 8, 0], np.int32)
    tgt = np.array([5, 5, 5, 1, 9], np.int32)
    via = np.array([[7, -1], [0, 9], [-1, 4], [8, 8], [-1, -1]], np.int32)
    forbid = np.array([[-1], [-1], [-1], [-1], [5]], np.int32)
    d, _ = orc.reach_via(n, topo["adj_off"], topo["adj"], region, src, np.ones(5, np.uint32), tgt, via, forbid)
    # 2->7->5: 5 + 2; 2->0->9->5: 2 + 9 + 4; via starting with -1 = none: 3;
    # 8->8->8->1: 7; a forbidden cut vertex on a path: none
    assert list(d) == [7, 15, 3, 7, -1]
    # cycle of 12: forbidding a vertex on the short arc forces the long one
    c = 12
    cyc = ports_topology([[(v - 1) % c, (v + 1) % c] for v in range(c)], [0] * c)
    d, _ = orc.reach_via(c, cyc["adj_off"], cyc["adj"], np.zeros(c, np.uint8), np.array([0, 0], np.int32),
                         np.ones(2, np.uint32), np.array([3, 3], np.int32), np.full((2, 1), -1, np.int32),
                         np.array([[-1], [2]], np.int32))
    assert list(d) == [3, c - 3]


def test_via_fat_tree(orc):
    k = 4
    topo = synth.fat_tree(k, 2)
    S = topo["S"]
    region = np.zeros(S, np.uint8)
    core = k * k  # first core switch
    # edge 0 (pod 0) -> core -> edge 2 (pod 1); same pod via core; every agg of pod 0 forbidden
    src = np.array([0, 0, 0], np.int32)
    tgt = np.array([k, 1, k], np.int32)
    via = np.array([[core], [core], [core]], np.int32)
    forbid = np.array([[-1, -1], [-1, -1], [k // 2, k // 2 + 1]], np.int32)
    d, err = orc.reach_via(S, topo["adj_off"], topo["adj"], region, src, np.ones(3, np.uint32), tgt, via, forbid)
    assert err == 0
    assert list(d) == [4, 4, -1]


def test_via_without_constraints_is_reach(orc):
    wl = synth.cfg1(0)
    Q = wl["src"].shape[0]
    want, _ = orc.reach(wl["V"], wl["adj_off"], wl["adj"], wl["region"], wl["src"], wl["allowed"], wl["target"])
    got, _ = orc.reach_via(wl["V"], wl["adj_off"], wl["adj"], wl["region"], wl["src"], wl["allowed"],
                           wl["target"], np.full((Q, 2), -1, np.int32), np.full((Q, 1), -1, np.int32))
    assert np.array_equal(got, want)


def test_via_malformed(orc):
    topo = line_topology(4, [0] * 4)
    d, err = orc.reach_via(4, topo["adj_off"], topo["adj"], np.zeros(4, np.uint8), np.array([0, 0], np.int32),
                           np.ones(2, np.uint32), np.array([3, 3], np.int32), np.array([[9], [-1]], np.int32),
                           np.array([[-1], [-7]], np.int32))
    assert err & orc.F_SWITCH
    assert list(d) == [-1, 3]  # a waypoint out of range has no path; a bad forbidden entry is ignored


# ---------------------------------------------------------------- verdict

def _one_network_intent(orc, visit, pexp, jmask=1, state=0):
    intents = np.zeros(1, synth.INTENT_DT)
    intents["kind"] = synth.KIND_NETWORK
    intents["sel_row"] = -1
    intents["trace_end"] = 1
    intents["allowed"] = 1
    expect = np.zeros(1, synth.EXPECT_DT)
    expect["dst_switch"] = -1
    expect["dst_port"] = -1
    expect["reach_q"] = -1
    tr = np.zeros(1, orc.TRACE_DT)
    tr["jmask"] = jmask
    tr["state"] = state
    pe = np.zeros(1, synth.PATH_EXPECT_DT)
    pe["must"], pe["forbid"] = pexp
    return intents, expect, tr, np.array([visit], np.uint32), pe


@pytest.mark.parametrize("visit,pexp,jmask,state,want", [
    (0b001, (0b001, 0b110), 1, 0, 0),   # waypoint seen, nothing forbidden
    (0b011, (0b001, 0b110), 1, 0, 8),   # forbidden switch visited
    (0b000, (0b001, 0b110), 1, 0, 9),   # waypoint missed
    (0b010, (0b001, 0b110), 1, 0, 8),   # both: the smaller code
    (0b010, (0b001, 0b110), 3, 0, 4),   # a leak comes first
    (0b010, (0b001, 0b110), 1, 2, 5),   # undelivered comes first
    (0b000, (0b000, 0b000), 1, 0, 0),   # no path constraints
])
def test_report_path_fixtures(orc, visit, pexp, jmask, state, want):
    intents, expect, tr, vis, pe = _one_network_intent(orc, visit, pexp, jmask, state)
    feas = np.zeros((0, 1), np.uint64)
    pss, reason, summ, err = orc.report(intents, feas, np.zeros(0, np.uint32), 1, tr, expect, np.zeros(0, np.int32),
                                        vis, pe)
    assert err == 0 and int(reason[0]) == want
    assert (int(pss[0]) & 1) == (want == 0)
    assert summ["counts"][synth.KIND_NETWORK][want] == 1


def test_report_paths_cfg1_invariants(orc):
    wl = synth.cfg1(0, paths=True)
    o = orc.run_workload(wl)
    _, visit, _ = _watch_trace(orc, wl, wl["watch"])
    d, _ = orc.reach_via(wl["V"], wl["adj_off"], wl["adj"], wl["region"], wl["src"], wl["allowed"], wl["target"],
                         wl["via"], wl["forbid"])
    pss, reason, summ, err = orc.report(wl["intents"], o["feasible"], o["popcnt"], wl["N"], o["traces"],
                                        wl["expect"], d, visit, wl["pexp"])
    assert err == 0
    it, pe = wl["intents"], wl["pexp"]
    plain = o["reason"] & 0x7F
    r = reason & 0x7F
    for i in range(it.shape[0]):
        if plain[i] != 0:  # path checks only add failures, with larger codes
            assert r[i] == plain[i]
            continue
        tr = range(it["trace_begin"][i], it["trace_end"][i])
        hit = any(int(visit[t]) & int(pe["forbid"][i]) for t in tr)
        miss = any((int(visit[t]) & int(pe["must"][i])) != int(pe["must"][i]) for t in tr)
        assert r[i] == (8 if hit else 9 if miss else 0)
    # a network intent passes its path checks only if a constrained walk exists
    for i in np.flatnonzero((it["kind"] & 2) != 0):
        if r[i] == 0:
            q = wl["expect"]["reach_q"][i]
            assert 0 <= d[q] <= min(int(o["traces"][t]["hops"]) for t in
                                    range(it["trace_begin"][i], it["trace_end"][i]))
