"""Parity of the HIP path (through the C ABI) with the CPU oracle, element
by element, on seeded inputs small enough for the oracle to finish in
seconds while spanning several tiles and ragged tails.  Everything here is
integer / bitset work: the bar is bit-exact equality, including the
data-error flags."""
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


def _same_traces(a, b):
    assert a.shape == b.shape
    for f in ("jmask", "last_switch", "last_port", "hops", "state"):
        bad = np.flatnonzero(a[f] != b[f])
        assert bad.size == 0, f"field {f}: first mismatch at trace {bad[0]}: gpu {a[bad[0]]} oracle {b[bad[0]]}"


def _same(a, b, what):
    a, b = np.asarray(a), np.asarray(b)
    assert a.shape == b.shape, (what, a.shape, b.shape)
    bad = np.argwhere(a != b)
    assert bad.size == 0, f"{what}: first mismatch at {tuple(bad[0])}: gpu {a[tuple(bad[0])]} oracle {b[tuple(bad[0])]}"


def _check_workload(g, orc, wl):
    gp = g.run_workload(wl)
    oo = orc.run_workload(wl)
    flags = 0
    if "feasible" in oo:
        _same(gp["feasible"], oo["feasible"], "feasible")
        _same(gp["popcnt"], oo["popcnt"], "popcnt")
        flags |= oo["sel_err"]
    if "traces" in oo:
        _same_traces(gp["traces"], oo["traces"])
        flags |= oo["trace_err"]
    if "reach" in oo:
        _same(gp["reach"], oo["reach"], "reach")
        flags |= oo["reach_err"]
    if "reason" in oo:
        _same(gp["reason"], oo["reason"], "reason")
        _same(gp["pass"], oo["pass"], "pass")
        for f in ("counts", "no_path"):
            _same(gp["summary"][f], oo["summary"][f], f)
        flags |= oo["report_err"]
    assert gp["flags"] == flags
    return gp, oo


@pytest.mark.parametrize("variant", ["rpath", "literal", "dense"])
def test_cfg1_end_to_end(g, orc, variant, trace_path):
    _check_workload(g, orc, synth.cfg1(0, variant))


@pytest.mark.parametrize("seed", [1, 2])
def test_combined_small(g, orc, seed):
    wl = synth.combined_workload(seed, 3000 + 37, 16, 8, 4, 700, 3001)
    gp, oo = _check_workload(g, orc, wl)
    r = oo["reason"] & 0x7F
    assert (r == 0).sum() > 0 and (r == 1).sum() > 0 and (r == 4).sum() > 0


def test_selectors_absent_labels_and_ragged(g, orc):
    wl = synth.selector_workload(5, 5000 + 37, 12, 700, card_choices=(2, 3, 16, 64, 200), absent_p=0.05)
    _check_workload(g, orc, wl)


def test_selectors_many_planes(g, orc):
    """About 3,000 value planes with a few absent labels: long In/NotIn
    programs and a ragged last word."""
    wl = synth.selector_workload(21, 2000 + 11, 12, 300, card_choices=(250,), absent_p=0.01)
    _check_workload(g, orc, wl)


def test_selectors_large_value_sets(g, orc):
    """In/NotIn sets with up to 200 values (beyond the generators' 1..4)."""
    rng = np.random.default_rng(7)
    N, L = 3000, 5
    cards = np.array([250, 255, 7, 130, 2])
    labels = synth.gen_labels(rng, N, cards, absent_p=0.1)
    I = 300
    k = rng.integers(1, 4, size=I)
    off = np.zeros(I + 1, np.int32)
    off[1:] = np.cumsum(k)
    preds = np.zeros(int(off[-1]), synth.PRED_DT)
    for p in range(preds.shape[0]):
        l = int(rng.integers(0, L))
        preds[p]["label"] = l
        preds[p]["op"] = int(rng.integers(0, 3))
        m = int(rng.integers(0, min(200, cards[l]) + 1))
        vals = rng.choice(255, size=m, replace=False)
        bm = [0, 0, 0, 0]
        for v in vals:
            bm[v >> 6] |= 1 << int(v & 63)
        preds[p]["vals"] = np.array(bm, np.uint64)
    fg, pg = g.selectors(labels, off, preds)
    fo, po, _ = orc.selectors(labels, off, preds)
    _same(fg, fo, "feasible")
    _same(pg, po, "popcnt")


def test_selectors_program_lengths(g, orc):
    """Rows whose compiled programs have every length from 0 to 40 entries:
    the empty program, the 8-entry group boundary, the 15-entry inline
    limit and the indirect programs beyond it.  Each row is one In/NotIn
    predicate of m values on a 128-value label (a program of min(m, 128 - m)
    entries), possibly followed by an Exists and a second small predicate;
    absent values make Exists cost one entry."""
    rng = np.random.default_rng(12)
    N, L = 2500 + 17, 3
    cards = np.array([128, 128, 5])
    labels = synth.gen_labels(rng, N, cards, absent_p=0.05)
    rows = []
    for m in range(0, 41):
        for extra in range(3):
            preds = []
            for op in (0, 1):
                row = [(0, op, rng.choice(128, size=m, replace=False))]
                if extra >= 1:
                    row.append((1, 2, []))
                if extra >= 2:
                    row.append((2, int(rng.integers(0, 2)), rng.choice(5, size=2, replace=False)))
                preds.append(row)
            rows.extend(preds)
    off = np.zeros(len(rows) + 1, np.int32)
    off[1:] = np.cumsum([len(r) for r in rows])
    preds = np.zeros(int(off[-1]), synth.PRED_DT)
    p = 0
    for row in rows:
        for lab, op, vals in row:
            bm = [0, 0, 0, 0]
            for v in vals:
                bm[int(v) >> 6] |= 1 << int(v & 63)
            preds[p]["label"] = lab
            preds[p]["op"] = op
            preds[p]["vals"] = np.array(bm, np.uint64)
            p += 1
    fg, pg = g.selectors(labels, off, preds)
    fo, po, err = orc.selectors(labels, off, preds)
    assert err == 0
    _same(fg, fo, "feasible")
    _same(pg, po, "popcnt")


# (W, ragged bits, output offset in words): odd and even widths whose rows
# are shifted onto 128-byte lines (W = 200, 263, 781, 1000), widths where
# the shift would cost a tile and is off (W = 128, 255), and outputs that
# start 8 and 24 bytes into a line
@pytest.mark.parametrize("W,ragged,offset", [(200, 0, 0), (263, 17, 1), (781, 63, 3), (1000, 5, 0), (128, 1, 1),
                                             (255, 0, 3)])
def test_selectors_line_shifted_rows(g, orc, W, ragged, offset):
    """Every bitset word written exactly once, at its place, with the
    guard words around the output untouched."""
    import torch

    import paper_2602_16100_amd as pc
    N = 64 * W - ragged
    wl = synth.selector_workload(30 + W, N, 10, 333)
    fo, po, _ = orc.selectors(wl["labels"], wl["pred_off"], wl["preds"])
    I = wl["pred_off"].shape[0] - 1
    guard = np.int64(0x5A5A5A5A5A5A5A5A)
    buf = torch.full((I * W + offset + 8,), int(guard), dtype=torch.int64, device="cuda")
    out = buf[offset:offset + I * W].view(I, W)
    f, p = pc.pc_eval_selectors(g.dev(wl["labels"]), g.dev(wl["pred_off"]), g.dev(wl["preds"]), feasible=out)
    torch.cuda.synchronize()
    _same(f.cpu().numpy().view(np.uint64), fo, "feasible")
    _same(p.cpu().numpy().view(np.uint32), po, "popcnt")
    b = buf.cpu().numpy()
    assert (b[:offset] == guard).all() and (b[offset + I * W:] == guard).all()


def test_selectors_malformed_flags(g, orc):
    import paper_2602_16100_amd as pc
    wl = synth.selector_workload(9, 777, 6, 40)
    preds = wl["preds"].copy()
    off = wl["pred_off"].copy()
    preds[3]["label"] = 99          # label >= L
    preds[10]["op"] = 7             # bad op
    preds[20]["rsv1"] = 1
    off[30] = off[31] + 5           # decreasing pair for row 29 / row 30
    ctx = pc.context()
    ctx.data_errors(clear=True)
    fg, pg = g.selectors(wl["labels"], off, preds)
    flags = ctx.data_errors(clear=True)
    fo, po, err = orc.selectors(wl["labels"], off, preds)
    _same(fg, fo, "feasible")
    _same(pg, po, "popcnt")
    assert flags == err and err & orc.F_PRED and err & orc.F_OFFSETS


@pytest.fixture(params=["buckets", "default", "walk"])
def trace_path(request, monkeypatch):
    """Force the level-synchronous bucketed path, the default switch-over,
    or the per-trace walk for every level."""
    if request.param == "buckets":
        monkeypatch.setenv("PC_TRACE_WALK_MAX", "0")
    elif request.param == "walk":
        monkeypatch.setenv("PC_TRACE_WALK_MAX", str(10**9))
    return request.param


@pytest.mark.parametrize("variant", ["rpath", "literal", "dense", "prefix"])
def test_trace_fat_tree_small(g, orc, variant, trace_path):
    wl = synth.trace_workload(3, 8, 4, 512, 20000, 24, 3000, variant=variant)
    _check_workload(g, orc, wl)


def test_trace_switches_without_rules(g, orc, trace_path):
    """Every fifth switch (pod and core switches alike) has an empty flow
    table: every lookup there is a table miss, so the traces that reach such
    a switch, at ingress or in transit, end there in MISS."""
    wl = synth.trace_workload(3, 8, 4, 512, 20000, 24, 3000, variant="rpath")
    ro = np.asarray(wl["rule_off"], np.int64)
    S = wl["S"]
    empty = np.zeros(S, bool)
    empty[::5] = True
    keep = [wl["rules"][ro[s]:ro[s + 1]] for s in range(S) if not empty[s]]
    off = np.zeros(S + 1, np.int32)
    off[1:] = np.cumsum([0 if empty[s] else ro[s + 1] - ro[s] for s in range(S)])
    wl.arrays["rule_off"] = off
    wl.arrays["rules"] = np.concatenate(keep)
    _, oo = _check_workload(g, orc, wl)
    tr = oo["traces"]
    ended = tr["last_switch"] >= 0
    at_empty = np.zeros(tr.shape[0], bool)
    at_empty[ended] = empty[tr["last_switch"][ended]]
    assert np.all(tr["state"][at_empty] == 2)   # MISS
    assert at_empty.sum() > 100 and (at_empty & (tr["hops"] > 0)).any()


def test_trace_prefix_tables_multi_slice(g, orc, trace_path):
    """Routing tables (destination prefixes of 16-32 bits, ports, source and
    protocol wildcarded): each switch filters on the key nibbles its own
    rules care about, not on the port bits; 2,048 rules per switch (4
    slices), many rules per destination, so many filter survivors."""
    wl = synth.trace_workload(8, 16, 8, 2048, 40000, 32, 20000, variant="prefix")
    _check_workload(g, orc, wl)


def test_trace_mixed_tables(g, orc, trace_path):
    """Switches whose tables mix i.i.d. care bits, destination prefixes and
    rules that care only about the protocol byte or nothing at all: the
    per-switch filter chunks differ from switch to switch."""
    wl = synth.trace_workload(9, 8, 4, 700, 20000, 24, 3000, variant="rpath")
    rules = wl["rules"].copy()
    ro = wl["rule_off"]
    rng = np.random.default_rng(5)
    for s in range(wl["S"]):
        seg = slice(ro[s], ro[s + 1])
        kind = s % 4
        if kind == 1:       # destination prefixes
            m = synth.prefix_masks(rng, ro[s + 1] - ro[s])
        elif kind == 2:     # protocol byte only, half of them
            m = np.zeros((ro[s + 1] - ro[s], 4), np.uint32)
            m[::2, 3] = 0xFF
        elif kind == 3:     # wildcard everything in every third rule
            m = rules["mask"][seg].copy()
            m[::3] = 0
        else:
            continue
        rules["mask"][seg] = m
        rules["value"][seg] &= m
    wl.arrays["rules"] = rules
    _check_workload(g, orc, wl)


def test_trace_multi_slice_and_big_buckets(g, orc, trace_path):
    """20,000 rules per switch (two 16,384-rule slices) and buckets larger
    than one 2,048-lookup tile."""
    wl = synth.trace_workload(4, 4, 2, 20000, 12000, 16, 2000)
    _check_workload(g, orc, wl)


def test_trace_ties_and_ttl(g, orc, trace_path):
    rng = np.random.default_rng(3)
    topo = synth.random_graph(rng, 9, 14, 2, 4)
    rule_off, rules, _ = synth.build_tables(rng, topo, 40, 0.03, prio="small", prio_range=3)
    T = 3000
    hdr = synth.random_keys(rng, T)
    ingress = rng.integers(0, 9, size=T).astype(np.int32)
    for ttl in (0, 1, 7, 255):
        tg = g.trace(9, topo["port_off"], topo["port_peer"], topo["jur"], rule_off, rules, hdr, ingress, ttl)
        to, _ = orc.trace(9, topo["port_off"], topo["port_peer"], topo["jur"], rule_off, rules, hdr, ingress, ttl)
        _same_traces(tg, to)


def test_trace_switches_with_many_ports(g, orc, trace_path):
    """A dense random graph (100 switches of 74-89 ports: most have link
    ports past the first 64, and every host port is past them) with mostly
    wildcard rules: traces wander through high ports, whose peers and
    jurisdictions the match epilogue takes from the port table rather than
    from its staged first 64 ports."""
    rng = np.random.default_rng(11)
    topo = synth.random_graph(rng, 100, 4000, 2, 8)
    rule_off, rules, _ = synth.build_tables(rng, topo, 40, 0.03, prio="small", prio_range=3)
    T = 4000
    hdr = synth.random_keys(rng, T)
    ingress = rng.integers(0, 100, size=T).astype(np.int32)
    tg = g.trace(100, topo["port_off"], topo["port_peer"], topo["jur"], rule_off, rules, hdr, ingress, 16)
    to, _ = orc.trace(100, topo["port_off"], topo["port_peer"], topo["jur"], rule_off, rules, hdr, ingress, 16)
    _same_traces(tg, to)
    egress = to["state"] == 0
    assert egress.sum() > 100 and np.all(to["last_port"][egress] >= 64)


def test_trace_malformed_flags(g, orc):
    import paper_2602_16100_amd as pc
    wl = synth.trace_workload(6, 4, 2, 64, 500, 8, 100)
    jur = wl["jur"].copy()
    jur[3] = 40
    peer = wl["port_peer"].copy()
    peer[5] = 9999
    rules = wl["rules"].copy()
    rules["action"][17] = 77
    ingress = wl["ingress"].copy()
    ingress[4] = -3
    ctx = pc.context()
    ctx.data_errors(clear=True)
    tg = g.trace(wl["S"], wl["port_off"], peer, jur, wl["rule_off"], rules, wl["hdr"], ingress, wl["ttl"])
    flags = ctx.data_errors(clear=True)
    to, err = orc.trace(wl["S"], wl["port_off"], peer, jur, wl["rule_off"], rules, wl["hdr"], ingress, wl["ttl"])
    _same_traces(tg, to)
    assert flags == err == (orc.F_JUR | orc.F_SWITCH | orc.F_ACTION)


@pytest.mark.parametrize("full_rows", [True, False])
def test_reach_small_graph_bitset(g, orc, full_rows):
    wl = synth.rgg_workload(4, 3000, 8, 200, mean_degree=6.0, full_rows=full_rows)
    _check_workload(g, orc, wl)


@pytest.mark.parametrize("V", [700, 1500, 2900, 4000, 5500, 6016, 6200])
def test_reach_bitset_sizes(g, orc, V):
    """The bitset BFS up to its largest LDS-resident graph (6,016 vertices)
    and just past it (the queue path), target mode and full rows."""
    for full_rows in (False, True):
        wl = synth.rgg_workload(V, V, 8, 130, mean_degree=7.0, full_rows=full_rows)
        _check_workload(g, orc, wl)


@pytest.mark.parametrize("deg", [7.0, 20.0, 40.0, 80.0])
def test_reach_bitset_lane_groups(g, orc, deg):
    """Mean degrees that select 4, 8, 16 and 32 lanes per frontier vertex."""
    for full_rows in (False, True):
        wl = synth.rgg_workload(int(deg), 1500, 8, 150, mean_degree=deg, full_rows=full_rows)
        _check_workload(g, orc, wl)


@pytest.mark.parametrize("full_rows", [True, False])
def test_reach_large_graph_queue(g, orc, full_rows):
    wl = synth.rgg_workload(5, 40000, 16, 40, mean_degree=5.0, full_rows=full_rows)
    _check_workload(g, orc, wl)


def test_reach_fat_tree_targets(g, orc):
    topo = synth.fat_tree(16, 6)
    rng = np.random.default_rng(1)
    Q = 1000
    src = rng.integers(0, topo["S"], size=Q).astype(np.int32)
    tgt = rng.integers(0, topo["S"], size=Q).astype(np.int32)
    allowed = rng.integers(0, 64, size=Q).astype(np.uint32)
    dg = g.reach(topo["S"], topo["adj_off"], topo["adj"], topo["jur"], src, allowed, tgt)
    do, _ = orc.reach(topo["S"], topo["adj_off"], topo["adj"], topo["jur"], src, allowed, tgt)
    _same(dg, do, "dist")
    assert (do >= 0).sum() > 100 and (do == -1).sum() > 100


@pytest.mark.parametrize("kind", ["asymmetric", "unsorted", "bad_offsets"])
def test_reach_targets_on_one_way_graphs(g, orc, kind):
    """Resolving a target one level early from its own adjacency list is
    exact only when the lists are symmetric: one-way entries, unsorted lists
    (which switch the shortcut off) and a vertex with invalid offsets (named
    by lists it cannot name back) must match the oracle's plain search."""
    wl = synth.rgg_workload(11, 1200, 4, 130, mean_degree=9.0, full_rows=False)
    adj_off, adj = wl["adj_off"].copy(), wl["adj"].copy()
    rng = np.random.default_rng(1)
    if kind == "asymmetric":
        for p in rng.choice(adj.shape[0], size=40, replace=False):
            adj[p] = int(rng.integers(0, wl["V"]))
        for u in range(wl["V"]):
            adj[adj_off[u]:adj_off[u + 1]] = np.sort(adj[adj_off[u]:adj_off[u + 1]])
    elif kind == "unsorted":
        for u in range(wl["V"]):
            adj[adj_off[u]:adj_off[u + 1]] = adj[adj_off[u]:adj_off[u + 1]][::-1]
    else:
        hub = int(np.argmax(np.diff(adj_off)))
        adj_off[hub + 1] = adj_off[hub] - 1 if adj_off[hub] > 0 else adj.shape[0] + 5
    dg = g.reach(wl["V"], adj_off, adj, wl["region"], wl["src"], wl["allowed"], wl["target"])
    do, _ = orc.reach(wl["V"], adj_off, adj, wl["region"], wl["src"], wl["allowed"], wl["target"])
    _same(dg, do, "dist")


def test_reach_malformed_flags(g, orc):
    import paper_2602_16100_amd as pc
    wl = synth.rgg_workload(2, 800, 4, 70, mean_degree=6.0, full_rows=False)
    adj = wl["adj"].copy()
    adj[11] = -5
    region = wl["region"].copy()
    region[2] = 33
    src = wl["src"].copy()
    src[1] = 10**6
    ctx = pc.context()
    ctx.data_errors(clear=True)
    dg = g.reach(wl["V"], wl["adj_off"], adj, region, src, wl["allowed"], wl["target"])
    flags = ctx.data_errors(clear=True)
    do, err = orc.reach(wl["V"], wl["adj_off"], adj, region, src, wl["allowed"], wl["target"])
    _same(dg, do, "dist")
    assert flags == err == (orc.F_GRAPH | orc.F_JUR | orc.F_SWITCH)


def test_report_malformed_intents(g, orc):
    wl = synth.cfg1(0)
    oo = orc.run_workload(wl)
    it = wl["intents"].copy()
    it[2]["kind"] = 9
    it[4]["trace_end"] = 99999
    it[5]["sel_row"] = -2
    pg, rg, sg = g.report(it, oo["feasible"], oo["popcnt"], wl["N"], oo["traces"], wl["expect"], oo["reach"])
    po, ro, so, err = orc.report(it, oo["feasible"], oo["popcnt"], wl["N"], oo["traces"], wl["expect"], oo["reach"])
    _same(rg, ro, "reason")
    _same(pg, po, "pass")
    _same(sg["counts"], so["counts"], "counts")


def test_selectors_plane_tables_past_2gib(g, orc):
    """8,000 labels over 3,000 nodes: the value-plane table (8,000 x 256
    possible values, 144 words each) passes 2 GiB, so the evaluator reads
    planes through 64-bit pointers instead of 32-bit buffer offsets."""
    wl = synth.selector_workload(41, 3000, 8000, 300, card_choices=(2, 3, 16, 64), absent_p=0.05)
    assert 8000 * 256 * 144 * 8 >= 1 << 31
    fg, pg = g.selectors(wl["labels"], wl["pred_off"], wl["preds"])
    fo, po, err = orc.selectors(wl["labels"], wl["pred_off"], wl["preds"])
    _same(fg, fo, "feasible")
    _same(pg, po, "popcnt")
    assert err == 0 and (po > 0).sum() > 100


def test_empty_inputs(g, orc):
    """N = 0, I = 0, T = 0, Q = 0 and V = 0 all return cleanly."""
    labels = np.zeros((0, 4), np.uint8)
    off = np.zeros(4, np.int32)
    preds = np.zeros(0, synth.PRED_DT)
    fg, pg = g.selectors(labels, off, preds)
    assert fg.shape == (3, 0) and list(pg) == [0, 0, 0]
    topo = synth.fat_tree(4, 2)
    tg = g.trace(topo["S"], topo["port_off"], topo["port_peer"], topo["jur"], np.zeros(topo["S"] + 1, np.int32),
                 np.zeros(0, synth.RULE_DT), np.zeros((0, 4), np.uint32), np.zeros(0, np.int32), 5)
    assert tg.shape == (0,)
    dg = g.reach(0, np.zeros(1, np.int32), np.zeros(0, np.int32), np.zeros(0, np.uint8), np.array([0], np.int32),
                 np.array([1], np.uint32), np.array([0], np.int32))
    assert list(dg) == [-1]


def test_determinism(g, orc):
    wl = synth.combined_workload(3, 2000, 8, 8, 4, 300, 999)
    a = g.run_workload(wl)
    b = g.run_workload(wl)
    for k in ("feasible", "popcnt", "reach", "reason", "pass"):
        _same(a[k], b[k], k)
    _same_traces(a["traces"], b["traces"])
