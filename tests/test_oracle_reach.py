"""Pins for the oracle's masked reachability (compliant-path existence and
hop distance inside the allowed-induced subgraph).

Pins: networkx and scipy unweighted shortest paths on the induced
subgraph, brute force over all simple paths on tiny graphs and every
region mask, closed forms (path graph, fat-tree), BFS-layer invariants.
"""
import itertools

import networkx as nx
import numpy as np
import pytest
from scipy.sparse import csr_matrix
from scipy.sparse.csgraph import shortest_path

import synth
from helpers import line_topology


def _induced(V, adj_off, adj, region, allowed):
    G = nx.Graph()
    ok = [v for v in range(V) if (allowed >> int(region[v])) & 1]
    G.add_nodes_from(ok)
    oks = set(ok)
    for u in ok:
        for p in range(adj_off[u], adj_off[u + 1]):
            v = int(adj[p])
            if v in oks:
                G.add_edge(u, v)
    return G


def _nx_row(V, G, s):
    row = np.full(V, -1, np.int64)
    if s in G:
        for v, d in nx.single_source_shortest_path_length(G, s).items():
            row[v] = d
    return row


def test_networkx_small_rgg(orc):
    wl = synth.rgg_workload(4, 3000, 8, 24, mean_degree=6.0)
    dist, err = orc.reach(wl["V"], wl["adj_off"], wl["adj"], wl["region"], wl["src"], wl["allowed"])
    assert err == 0
    for q in range(24):
        G = _induced(wl["V"], wl["adj_off"], wl["adj"], wl["region"], int(wl["allowed"][q]))
        assert np.array_equal(dist[q], _nx_row(wl["V"], G, int(wl["src"][q])))


def test_scipy_all_allowed(orc):
    wl = synth.rgg_workload(6, 2000, 4, 10, mean_degree=5.0)
    allowed = np.full(10, 0xF, np.uint32)
    dist, _ = orc.reach(wl["V"], wl["adj_off"], wl["adj"], wl["region"], wl["src"], allowed)
    V = wl["V"]
    A = csr_matrix((np.ones(wl["adj"].shape[0]), wl["adj"], wl["adj_off"]), shape=(V, V))
    D = shortest_path(A, unweighted=True, indices=wl["src"])
    D = np.where(np.isinf(D), -1, D).astype(np.int64)
    assert np.array_equal(dist, D)


def test_brute_force_simple_paths(orc):
    """Every graph on 6 vertices from a random family, every region mask:
    distance = length of the shortest simple path through allowed vertices."""
    rng = np.random.default_rng(2)
    for g in range(25):
        V = 6
        edges = [(u, v) for u, v in itertools.combinations(range(V), 2) if rng.random() < 0.4]
        nbr = [[] for _ in range(V)]
        for u, v in edges:
            nbr[u].append(v)
            nbr[v].append(u)
        adj_off = np.zeros(V + 1, np.int32)
        adj = []
        for u in range(V):
            adj.extend(sorted(nbr[u]))
            adj_off[u + 1] = len(adj)
        adj = np.array(adj, np.int32)
        region = rng.integers(0, 3, size=V).astype(np.uint8)
        for mask in range(8):
            src = np.arange(V, dtype=np.int32)
            dist, _ = orc.reach(V, adj_off, adj, region, src, np.full(V, mask, np.uint32))
            for s in range(V):
                for t in range(V):
                    ok = lambda x: (mask >> int(region[x])) & 1
                    best = -1
                    if ok(s) and ok(t):
                        if s == t:
                            best = 0
                        else:
                            mids = [x for x in range(V) if x not in (s, t) and ok(x)]
                            E = set(edges) | {(b, a) for a, b in edges}
                            for k in range(len(mids) + 1):
                                for perm in itertools.permutations(mids, k):
                                    path = (s,) + perm + (t,)
                                    if all((path[i], path[i + 1]) in E for i in range(len(path) - 1)):
                                        best = len(path) - 1
                                        break
                                if best >= 0:
                                    break
                    assert dist[s, t] == best, (g, mask, s, t)


def test_path_graph_closed_form(orc):
    V = 50
    topo = line_topology(V, [0] * V)
    src = np.array([0, 17, 49], np.int32)
    dist, _ = orc.reach(V, topo["adj_off"], topo["adj"], topo["jur"], src, np.ones(3, np.uint32))
    for k, s in enumerate(src):
        assert np.array_equal(dist[k], np.abs(np.arange(V) - s))


@pytest.mark.parametrize("k", [4, 8])
def test_fat_tree_closed_forms(orc, k):
    topo = synth.fat_tree(k, 4)
    S, h = topo["S"], k // 2
    edges = [p * k + e for p in range(k) for e in range(h)]
    region = np.zeros(S, np.uint8)
    region[k * k:] = 1                                   # cores in region 1, pods in region 0
    src = np.array(edges, np.int32)
    d_all, _ = orc.reach(S, topo["adj_off"], topo["adj"], region, src, np.full(len(src), 3, np.uint32))
    d_pod, _ = orc.reach(S, topo["adj_off"], topo["adj"], region, src, np.full(len(src), 1, np.uint32))
    for i, s in enumerate(edges):
        for t in edges:
            same_pod = s // k == t // k
            want = 0 if s == t else (2 if same_pod else 4)
            assert d_all[i, t] == want
            assert d_pod[i, t] == (want if same_pod else -1)
        assert np.all(d_pod[i, k * k:] == -1)


def test_targets_and_disallowed_source(orc):
    wl = synth.rgg_workload(9, 1500, 6, 40, mean_degree=6.0, full_rows=False)
    full, _ = orc.reach(wl["V"], wl["adj_off"], wl["adj"], wl["region"], wl["src"], wl["allowed"])
    tgt, _ = orc.reach(wl["V"], wl["adj_off"], wl["adj"], wl["region"], wl["src"], wl["allowed"], wl["target"])
    assert np.array_equal(tgt, full[np.arange(40), wl["target"]])
    bad = wl["allowed"] & ~np.left_shift(np.uint32(1), wl["region"][wl["src"]].astype(np.uint32))
    full2, _ = orc.reach(wl["V"], wl["adj_off"], wl["adj"], wl["region"], wl["src"], bad)
    assert np.all(full2 == -1)


def test_bfs_layer_invariants(orc):
    wl = synth.rgg_workload(12, 20000, 16, 16)
    dist, _ = orc.reach(wl["V"], wl["adj_off"], wl["adj"], wl["region"], wl["src"], wl["allowed"])
    adj_off, adj, region = wl["adj_off"], wl["adj"], wl["region"]
    for q in range(16):
        A = int(wl["allowed"][q])
        d = dist[q]
        assert d[wl["src"][q]] == 0
        for v in np.flatnonzero(d >= 0):
            assert (A >> int(region[v])) & 1
            nb = adj[adj_off[v]:adj_off[v + 1]]
            okn = nb[((A >> region[nb].astype(np.int64)) & 1) == 1]
            assert np.all(d[okn] >= 0)                         # no reached vertex has an unreached allowed neighbour
            assert np.all(np.abs(d[okn] - d[v]) <= 1)          # layers differ by at most one across an edge
            if d[v] > 0:
                assert np.any(d[okn] == d[v] - 1)              # a parent one layer up


def test_malformed_graph(orc):
    topo = line_topology(4, [0, 0, 0, 0])
    adj = topo["adj"].copy()
    adj[0] = 99
    region = np.array([0, 0, 40, 0], np.uint8)
    dist, err = orc.reach(4, topo["adj_off"], adj, region, np.array([1, 9], np.int32), np.ones(2, np.uint32))
    assert err & orc.F_JUR and err & orc.F_SWITCH
    assert list(dist[0]) == [1, 0, -1, -1] and np.all(dist[1] == -1)
    dist, err = orc.reach(4, topo["adj_off"], adj, region, np.array([0], np.int32), np.ones(1, np.uint32))
    assert err & orc.F_GRAPH and list(dist[0]) == [0, -1, -1, -1]
