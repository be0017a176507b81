"""Pins of the CPU oracle's path synthesis (minimum-weight walks through
allowed, non-forbidden switches via ordered waypoints, and one exact-match
rule per switch of the walk).

The oracle is checked against things it does not compute itself:
- networkx: for each leg, every minimum-weight path of the usable subgraph
  is enumerated (all_shortest_paths) and the expected path is the
  lexicographically smallest one read from its end; lengths against
  networkx's BFS / Dijkstra;
- the separately pinned trace oracle: the compiled rules, installed into
  per-switch tables, carry each request's key from its source to an
  EGRESS at the target's host port along exactly the synthesized walk;
- closed forms on a path graph, a cycle and a fat-tree; failure cases.
"""
import networkx as nx
import numpy as np
import pytest

import synth


def _usable_graph(topo, weight, A, forbid):
    S = topo["S"]
    jur = topo["jur"]
    ok = [(int(jur[v]) < 32 and (A >> int(jur[v])) & 1) and v not in forbid for v in range(S)]
    G = nx.DiGraph()
    G.add_nodes_from(v for v in range(S) if ok[v])
    po, pp = topo["port_off"], topo["port_peer"]
    for u in range(S):
        if not ok[u]:
            continue
        for p in range(po[u], po[u + 1]):
            v = int(pp[p])
            w = 1 if weight is None else int(weight[p])
            if v < 0 or not ok[v] or w == 0:
                continue
            if not G.has_edge(u, v) or G[u][v]["w"] > w:
                G.add_edge(u, v, w=w)
    return G


def _expected_walk(topo, weight, A, stops, forbid):
    G = _usable_graph(topo, weight, A, set(forbid))
    walk = [stops[0]]
    for s, t in zip(stops[:-1], stops[1:]):
        if s not in G or t not in G or not nx.has_path(G, s, t):
            return None
        paths = list(nx.all_shortest_paths(G, s, t, weight=None if weight is None else "w"))
        best = min(paths, key=lambda p: p[::-1])
        walk.extend(best[1:])
    return walk


def _run(orc, topo, req, weight=None, max_hops=40, prio=1000):
    return orc.synthesize(topo["S"], topo["port_off"], topo["port_peer"], topo["jur"], req["src"], req["target"],
                          req["allowed"], req["via"], req["forbid"], req["key"], req["out_port"], prio, max_hops,
                          weight=weight)


@pytest.mark.parametrize("weighted", [False, True])
@pytest.mark.parametrize("kind", ["random", "fat_tree"])
def test_walks_against_networkx(orc, kind, weighted):
    rng = np.random.default_rng(3)
    topo = synth.random_graph(rng, 40, 70, 2, 4) if kind == "random" else synth.fat_tree(6, 3)
    weight = synth.port_weights(5, topo["port_peer"].shape[0], 6) if weighted else None
    req = synth.synthesis_requests(1, topo, 150, Kv=2, Kf=3)
    hops, path, rules, err = _run(orc, topo, req, weight)
    assert err == 0
    n_ok = 0
    for q in range(150):
        vq = req["via"][q].tolist()
        vq = vq[:vq.index(-1)] if -1 in vq else vq  # the list ends at its first -1
        stops = [int(req["src"][q])] + vq + [int(req["target"][q])]
        forbid = [int(v) for v in req["forbid"][q] if v >= 0]
        want = _expected_walk(topo, weight, int(req["allowed"][q]), stops, forbid)
        if want is None:
            assert hops[q] == -1 and (path[q] == -1).all()
            continue
        n_ok += 1
        assert hops[q] == len(want) - 1, q
        assert path[q, :len(want)].tolist() == want, q
        assert (path[q, len(want):] == -1).all()
    assert 0 < n_ok < 150


@pytest.mark.parametrize("weighted", [False, True])
def test_rules_realise_the_walk(orc, weighted):
    """Install the synthesized rules of every walk that repeats no switch
    and trace each request's key from its source: EGRESS at the target's
    host port, the walk's hop count, only allowed jurisdictions, and the
    walk's switches (waypoints in order)."""
    topo = synth.fat_tree(8, 4)
    weight = synth.port_weights(2, topo["port_peer"].shape[0]) if weighted else None
    Q = 300
    req = synth.synthesis_requests(3, topo, Q, Kv=1, Kf=2)
    hops, path, rules, err = _run(orc, topo, req, weight, max_hops=24)
    assert err == 0
    # a walk that passes a switch twice cannot be realised by rules that
    # match the 5-tuple only (both visits would need their own action)
    simple = np.array([h >= 0 and len(set(p[:h + 1])) == h + 1 for h, p in zip(hops, path)])
    ok = np.flatnonzero(simple)
    assert ok.size > 100 and (hops >= 0).sum() > ok.size
    S = topo["S"]
    per = [[] for _ in range(S)]
    for q in ok:
        for k in range(hops[q] + 1):
            per[path[q, k]].append(rules[q, k])
    rule_off = np.zeros(S + 1, np.int32)
    rule_off[1:] = np.cumsum([len(x) for x in per])
    table = np.array([r for x in per for r in x], synth.RULE_DT)
    out, visit, terr = orc.trace(S, topo["port_off"], topo["port_peer"], topo["jur"], rule_off, table,
                                 req["key"][ok], req["src"][ok], 255,
                                 watch=np.where(path[ok] >= 0, path[ok], -1)[:, :32])
    assert terr == 0
    assert (out["state"] == orc.EGRESS).all()
    assert np.array_equal(out["last_switch"], req["target"][ok])
    assert np.array_equal(out["last_port"].astype(np.int32), req["out_port"][ok])
    assert np.array_equal(out["hops"].astype(np.int32), hops[ok])
    assert ((out["jmask"] & ~req["allowed"][ok]) == 0).all()
    slots = np.minimum(hops[ok] + 1, 32)
    assert np.array_equal(visit, ((np.uint64(1) << slots.astype(np.uint64)) - np.uint64(1)).astype(np.uint32))
    # rules: exact match on the 104 key bits, the given priority
    r = rules[ok, 0]
    assert (r["mask"][:, :3] == 0xFFFFFFFF).all() and (r["mask"][:, 3] == 0xFF).all()
    assert (r["priority"] == 1000).all() and np.array_equal(r["value"], req["key"][ok])


def _line(n, hosts=1):
    po = np.zeros(n + 1, np.int32)
    peers = []
    for v in range(n):
        nb = [u for u in (v - 1, v + 1) if 0 <= u < n]
        peers.extend(nb + [-1] * hosts)
        po[v + 1] = len(peers)
    return po, np.array(peers, np.int32)


def test_closed_forms(orc):
    n = 10
    po, pp = _line(n)
    region = np.zeros(n, np.uint8)

    def one(s, t, via=(-1,), forbid=(-1,), out_port=None, max_hops=40, A=1, weight=None):
        op = out_port if out_port is not None else (1 if t in (0, n - 1) else 2)
        return orc.synthesize(n, po, pp, region, np.array([s], np.int32), np.array([t], np.int32),
                              np.array([A], np.uint32), np.array([via], np.int32), np.array([forbid], np.int32),
                              np.zeros((1, 4), np.uint32), np.array([op], np.int32), 7, max_hops, weight=weight)

    h, p, r, e = one(0, 9)
    assert e == 0 and h[0] == 9 and p[0, :10].tolist() == list(range(10))
    assert r[0, :9]["action"].tolist() == [0] + [1] * 8 and r[0, 9]["action"] == 1
    h, p, r, e = one(2, 2)
    assert h[0] == 0 and p[0, 0] == 2 and r[0, 0]["action"] == 2
    h, p, r, e = one(0, 9, via=(7, 3))  # 0 -> 7 -> 3 -> 9: 7 + 4 + 6 links
    assert h[0] == 17 and p[0, :18].tolist() == list(range(8)) + [6, 5, 4, 3] + list(range(4, 10))
    h, p, r, e = one(0, 9, forbid=(5,))
    assert h[0] == -1 and (p[0] == -1).all() and (r[0]["priority"] == 0).all()
    h, p, r, e = one(0, 9, max_hops=8)
    assert h[0] == -1
    h, p, r, e = one(0, 9, A=2)  # region 0 not allowed
    assert h[0] == -1
    h, p, r, e = one(0, 9, out_port=5)  # switch 9 has 2 ports
    assert h[0] == -1 and e == 4  # F_ACTION
    # a cycle 0..7: forbidding switch 1 forces the long arc 0 -> 7 -> ... -> 2
    m = 8
    po = np.arange(0, 3 * m + 1, 3, dtype=np.int32)
    pp = np.array([[(v - 1) % m, (v + 1) % m, -1] for v in range(m)], np.int32).ravel()
    h, p, r, e = orc.synthesize(m, po, pp, np.zeros(m, np.uint8), np.array([0, 0], np.int32),
                                np.array([2, 4], np.int32), np.array([1, 1], np.uint32),
                                np.array([[-1], [-1]], np.int32), np.array([[1], [-1]], np.int32),
                                np.zeros((2, 4), np.uint32), np.array([2, 2], np.int32), 1, 20)
    assert h.tolist() == [6, 4]
    assert p[0, :7].tolist() == [0, 7, 6, 5, 4, 3, 2]
    # both arcs to 4 have 4 links: the smaller predecessors read from the end win (3, 2, 1)
    assert p[1, :5].tolist() == [0, 1, 2, 3, 4]


def test_weights_pick_the_light_parallel_port(orc):
    """Two parallel links 0 -> 1 of weights 5 and 2: the rule uses the
    lighter; a heavy direct link loses to a lighter two-link detour."""
    po = np.array([0, 3, 6, 8], np.int32)
    pp = np.array([1, 1, 2, 0, 0, 2, 0, 1], np.int32)
    w = np.array([5, 2, 9, 1, 1, 3, 9, 3], np.uint32)
    h, p, r, e = orc.synthesize(3, po, pp, np.zeros(3, np.uint8), np.array([0, 0], np.int32),
                                np.array([1, 2], np.int32), np.array([1, 1], np.uint32),
                                np.full((2, 1), -1, np.int32), np.full((2, 1), -1, np.int32),
                                np.zeros((2, 4), np.uint32), np.array([0, 0], np.int32), 1, 5, weight=w)
    assert e == 0
    assert h.tolist() == [1, 2]
    assert r[0, 0]["action"] == 1
    assert p[1, :3].tolist() == [0, 1, 2] and r[1, 0]["action"] == 1 and r[1, 1]["action"] == 2


def test_distance_range(orc):
    """Leg distances are sums below 2^31 - 1 (the library's reading: the
    paper gives no range): a target at distance 2^31 - 2 is reached, one at
    2^31 - 1 or beyond is not, and a link of weight 2^31 - 1 or more is never
    taken, so a light detour wins over it."""
    big = (1 << 31) - 1

    def leg(po, pp, w, s, t):
        n = po.shape[0] - 1
        return orc.synthesize(n, po, pp, np.zeros(n, np.uint8), np.array([s], np.int32), np.array([t], np.int32),
                              np.array([1], np.uint32), np.full((1, 1), -1, np.int32), np.full((1, 1), -1, np.int32),
                              np.zeros((1, 4), np.uint32), np.array([0], np.int32), 1, 10,
                              weight=np.array(w, np.uint32))
    # a line 0 - 1 - 2: ports 0 -> 1, 1 -> 0, 1 -> 2, 2 -> 1
    po = np.array([0, 1, 3, 4], np.int32)
    pp = np.array([1, 0, 2, 1], np.int32)
    h, p, r, e = leg(po, pp, [big - 2, 1, 1, 1], 0, 2)  # 2^31 - 2
    assert e == 0 and h[0] == 2 and p[0, :3].tolist() == [0, 1, 2]
    h, p, r, e = leg(po, pp, [big - 2, 1, 2, 1], 0, 2)  # 2^31 - 1
    assert e == 0 and h[0] == -1
    h, p, r, e = leg(po, pp, [big - 2, 1, 2, 1], 0, 1)  # the first link alone, 2^31 - 3
    assert h[0] == 1
    for w01 in (big, big + 1, (1 << 32) - 1):
        h, p, r, e = leg(po, pp, [w01, 1, 1, 1], 0, 1)
        assert e == 0 and h[0] == -1, w01
    # 0 -> 3 directly at 2^31, or 0 -> 1 -> 2 -> 3 at 5 per link
    po = np.array([0, 2, 4, 6, 8], np.int32)
    pp = np.array([3, 1, 0, 2, 1, 3, 2, 0], np.int32)
    h, p, r, e = leg(po, pp, [1 << 31, 5, 5, 5, 5, 5, 5, 5], 0, 3)
    assert e == 0 and h[0] == 3 and p[0, :4].tolist() == [0, 1, 2, 3] and r[0, 0]["action"] == 1
    h, p, r, e = leg(po, pp, [7, 5, 5, 5, 5, 5, 5, 5], 0, 3)  # a light direct link wins
    assert h[0] == 1 and r[0, 0]["action"] == 0


def test_malformed_inputs(orc):
    topo = synth.fat_tree(4, 2)
    req = synth.synthesis_requests(0, topo, 20, Kv=1, Kf=1)
    pp = topo["port_peer"].copy()
    pp[3] = 999
    region = topo["jur"].copy()
    region[5] = 40
    w = np.ones(pp.shape[0], np.uint32)
    w[7] = 0
    via = req["via"].copy()
    via[0, 0] = -5
    src = req["src"].copy()
    src[1] = 1 << 20
    out_port = req["out_port"].copy()
    out_port[2] = 77
    h, p, r, e = orc.synthesize(topo["S"], topo["port_off"], pp, region, src, req["target"], req["allowed"],
                                via, req["forbid"], req["key"], out_port, 1, 20, weight=w)
    assert e == 8 | 16 | 32 | 4  # SWITCH | JUR | GRAPH | ACTION
    assert h[0] == -1 and h[1] == -1 and h[2] == -1


@pytest.mark.parametrize("weighted", [False, True])
def test_parallel_links_of_equal_weight_use_the_lowest_port(orc, weighted):
    """Switch 0 has three links to switch 1 (ports 0, 1, 2) of equal weight
    and a host port; the compiled rule forwards on port 0."""
    po = np.array([0, 4, 8], np.int32)
    pp = np.array([1, 1, 1, -1, 0, 0, 0, -1], np.int32)
    w = np.array([4, 4, 4, 1, 4, 4, 4, 1], np.uint32) if weighted else None
    h, p, r, e = orc.synthesize(2, po, pp, np.zeros(2, np.uint8), np.array([0, 1], np.int32),
                                np.array([1, 0], np.int32), np.array([1, 1], np.uint32),
                                np.full((2, 1), -1, np.int32), np.full((2, 1), -1, np.int32),
                                np.zeros((2, 4), np.uint32), np.array([3, 3], np.int32), 1, 5, weight=w)
    assert e == 0 and h.tolist() == [1, 1]
    assert r[:, 0]["action"].tolist() == [0, 0] and r[:, 1]["action"].tolist() == [3, 3]
