"""Parity of pc_synthesize_paths (through the C ABI) with the CPU oracle:
hop counts, walks and the 40-byte compiled rules, bit-exact, plus the
data-error word; on random graphs and fat-trees, BFS and weighted, with
waypoints, forbidden switches and every failure case.  End to end: the
synthesized rules of simple walks, installed as flow tables, are traced by
pc_trace_flows to EGRESS along exactly the synthesized walks."""
import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def g():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import gpu_run
    return gpu_run


def _same(a, b, what):
    a, b = np.asarray(a), np.asarray(b)
    assert a.shape == b.shape, (what, a.shape, b.shape)
    bad = np.argwhere(a != b)
    assert bad.size == 0, f"{what}: first mismatch at {tuple(bad[0])}: gpu {a[tuple(bad[0])]} oracle {b[tuple(bad[0])]}"


def _check(g, orc, V, port_off, port_peer, region, req, prio, max_hops, weight=None, n_ports=None):
    args = (V, port_off, port_peer, region, req["src"], req["target"], req["allowed"], req["via"], req["forbid"],
            req["key"], req["out_port"], prio, max_hops)
    hg, pg, rg, eg = g.synthesize(*args, weight=weight, n_ports=n_ports)
    ho, po, ro, eo = orc.synthesize(*args, weight=weight, n_ports=n_ports)
    _same(hg, ho, "hops")
    _same(pg, po, "path")
    _same(rg.view(np.uint8).reshape(rg.shape[0], rg.shape[1] * 40),
          ro.view(np.uint8).reshape(ro.shape[0], ro.shape[1] * 40), "rules")
    assert eg == eo, (eg, eo)
    return ho, po, ro


@pytest.mark.parametrize("weighted", [False, True])
@pytest.mark.parametrize("kind,Kv,Kf", [("random", 0, 0), ("random", 2, 3), ("fat_tree", 1, 2), ("fat_tree", 3, 5)])
def test_synthesis_parity(g, orc, kind, Kv, Kf, weighted):
    rng = np.random.default_rng(11)
    topo = synth.random_graph(rng, 300, 700, 2, 6) if kind == "random" else synth.fat_tree(12, 6)
    weight = synth.port_weights(4, topo["port_peer"].shape[0], 9) if weighted else None
    req = synth.synthesis_requests(5, topo, 700, Kv=max(Kv, 1), Kf=max(Kf, 1))
    if Kv == 0:
        req["via"] = np.full((700, 1), -1, np.int32)
    if Kf == 0:
        req["forbid"] = np.full((700, 1), -1, np.int32)
    ho, _, _ = _check(g, orc, topo["S"], topo["port_off"], topo["port_peer"], topo["jur"], req, 4321, 40, weight)
    assert (ho >= 0).sum() > 100 and (ho == -1).sum() > 0


@pytest.mark.parametrize("kind", ["random", "fat_tree"])
def test_synthesis_huge_weights(g, orc, kind):
    """Link weights up to 2^32 - 1, so that legs cross the 2^31 - 1 distance
    bound (beyond it a switch is unreachable) and 64-bit sums would differ from
    32-bit ones."""
    rng = np.random.default_rng(21)
    topo = synth.random_graph(rng, 300, 700, 2, 6) if kind == "random" else synth.fat_tree(8, 4)
    n = topo["port_peer"].shape[0]
    choices = np.array([1, 2, 7, 1 << 28, 1 << 29, (1 << 30) - 1, 1 << 30, (1 << 31) - 3, (1 << 31) - 2,
                        (1 << 31) - 1, 1 << 31, (1 << 32) - 1], np.uint64)
    weight = choices[rng.integers(0, choices.shape[0], n)].astype(np.uint32)
    req = synth.synthesis_requests(7, topo, 600, Kv=1, Kf=1)
    ho, _, _ = _check(g, orc, topo["S"], topo["port_off"], topo["port_peer"], topo["jur"], req, 99, 40, weight)
    assert (ho >= 0).sum() > 10 and (ho == -1).sum() > 10


def test_synthesis_max_hops_and_tiny_budgets(g, orc):
    topo = synth.fat_tree(8, 4)
    req = synth.synthesis_requests(6, topo, 400, Kv=2, Kf=1)
    for max_hops in (0, 1, 2, 4, 7, 255):
        _check(g, orc, topo["S"], topo["port_off"], topo["port_peer"], topo["jur"], req, 7, max_hops)


def test_synthesis_largest_graph(g, orc):
    """A random graph at the size limit (12,288 switches): the LDS state of
    one request at its largest."""
    rng = np.random.default_rng(2)
    topo = synth.random_graph(rng, 12288, 30000, 1, 3)
    req = synth.synthesis_requests(9, topo, 64, Kv=1, Kf=2)
    ho, _, _ = _check(g, orc, topo["S"], topo["port_off"], topo["port_peer"], topo["jur"], req, 1, 255,
                      synth.port_weights(1, topo["port_peer"].shape[0]))
    assert (ho > 0).any()


def test_synthesis_malformed(g, orc):
    topo = synth.fat_tree(6, 3)
    req = synth.synthesis_requests(0, topo, 60, Kv=1, Kf=1)
    pp = topo["port_peer"].copy()
    pp[3] = 999
    pp[10] = -7
    region = topo["jur"].copy()
    region[5] = 40
    w = np.ones(pp.shape[0], np.uint32)
    w[7] = 0
    req["via"][0, 0] = -5
    req["src"][1] = 1 << 20
    req["target"][2] = -3
    req["out_port"][3] = 77
    req["forbid"][4, 0] = 4000
    po = topo["port_off"].copy()
    po[9] = po[10] + 1  # a bad offset pair for switch 9 (and 8)
    _check(g, orc, topo["S"], po, pp, region, req, 1, 20, weight=w)


def test_synthesis_empty(g, orc):
    topo = synth.fat_tree(4, 2)
    req = synth.synthesis_requests(0, topo, 3, Kv=1, Kf=1)
    empty = {k: v[:0] for k, v in req.items()}
    _check(g, orc, topo["S"], topo["port_off"], topo["port_peer"], topo["jur"], empty, 1, 10)
    # no switches: every request fails (its endpoints are out of range)
    _check(g, orc, 0, np.zeros(1, np.int32), np.zeros(0, np.int32), np.zeros(0, np.uint8), req, 1, 10)


@pytest.mark.parametrize("weighted", [False, True])
def test_synthesized_rules_deliver_on_the_gpu(g, orc, weighted):
    """The compiled rules of every walk that repeats no switch, installed as
    the switches' flow tables and traced on the GPU: EGRESS at the target's
    host port after exactly the walk's links, inside the allowed
    jurisdictions."""
    topo = synth.fat_tree(16, 8)
    weight = synth.port_weights(8, topo["port_peer"].shape[0]) if weighted else None
    Q = 3000
    req = synth.synthesis_requests(12, topo, Q, Kv=1, Kf=2)
    hops, path, rules, err = g.synthesize(topo["S"], topo["port_off"], topo["port_peer"], topo["jur"], req["src"],
                                          req["target"], req["allowed"], req["via"], req["forbid"], req["key"],
                                          req["out_port"], 900, 32, weight=weight)
    assert err == 0
    simple = np.array([h >= 0 and len(set(p[:h + 1])) == h + 1 for h, p in zip(hops, path)])
    ok = np.flatnonzero(simple)
    assert ok.size > 1000
    S = topo["S"]
    sw = path[ok].ravel()
    rl = rules[ok].ravel()
    live = sw >= 0
    sw, rl = sw[live], rl[live]
    order = np.argsort(sw, kind="stable")
    sw, rl = sw[order], rl[order]
    rule_off = np.zeros(S + 1, np.int32)
    rule_off[1:] = np.cumsum(np.bincount(sw, minlength=S))
    tr = g.trace(S, topo["port_off"], topo["port_peer"], topo["jur"], rule_off, rl, req["key"][ok],
                 req["src"][ok], 255)
    assert (tr["state"] == 0).all()
    assert np.array_equal(tr["last_switch"], req["target"][ok])
    assert np.array_equal(tr["last_port"].astype(np.int32), req["out_port"][ok])
    assert np.array_equal(tr["hops"].astype(np.int32), hops[ok])
    assert ((tr["jmask"] & ~req["allowed"][ok]) == 0).all()
