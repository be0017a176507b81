"""Seeded synthetic inputs for the cross-layer compliance checker.

This module is test and benchmark infrastructure.  It builds clusters
(node labels), selector intents, switch topologies, flow tables, packet
headers, reachability queries and per-intent records, and nothing else:
it never evaluates a selector, matches a rule, walks a trace or runs a
search.  Both the CPU oracle and the GPU library consume exactly the
arrays produced here.

Record layouts (little-endian, packed as listed) are the C ABI's:

  pred    40 B  {u16 label, u8 op, u8 rsv0, u32 rsv1, u64 vals[4]}
  rule    40 B  {u32 value[4], u32 mask[4], u16 priority, u16 action, u32 rsv}
  key     16 B  u32[4] = {src_ip, dst_ip, sport<<16 | dport, proto}
  intent  32 B  {u8 kind, u8 pad[3], i32 sel_row, i32 src_node, i32 dst_node,
                 i32 trace_begin, i32 trace_end, u32 allowed, u32 pad2}
  expect  12 B  {i32 dst_switch, i32 dst_port, i32 reach_q}
  pexp     8 B  {u32 must, u32 forbid}   (masks over a trace's watch slots)

The workload recipes follow the paper's system model (labelled nodes,
a labelled switch graph, flow rules compiled per hop along a chosen
path; Sec. "Formal Model and Satisfaction" and "Network orchestration")
at the five benchmark scales; every free choice is a named parameter.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

# ---------------------------------------------------------------- records
PRED_DT = np.dtype([("label", "<u2"), ("op", "u1"), ("rsv0", "u1"),
                    ("rsv1", "<u4"), ("vals", "<u8", (4,))])
RULE_DT = np.dtype([("value", "<u4", (4,)), ("mask", "<u4", (4,)),
                    ("priority", "<u2"), ("action", "<u2"), ("rsv", "<u4")])
INTENT_DT = np.dtype([("kind", "u1"), ("pad", "u1", (3,)), ("sel_row", "<i4"),
                      ("src_node", "<i4"), ("dst_node", "<i4"),
                      ("trace_begin", "<i4"), ("trace_end", "<i4"),
                      ("allowed", "<u4"), ("pad2", "<u4")])
EXPECT_DT = np.dtype([("dst_switch", "<i4"), ("dst_port", "<i4"), ("reach_q", "<i4")])
assert PRED_DT.itemsize == 40 and RULE_DT.itemsize == 40
assert INTENT_DT.itemsize == 32 and EXPECT_DT.itemsize == 12

OP_IN, OP_NOTIN, OP_EXISTS = 0, 1, 2
OP_DOESNOTEXIST, OP_GT, OP_LT = 3, 4, 5
ABSENT = 0xFF
DROP = 0xFFFF
KIND_COMPUTE, KIND_NETWORK, KIND_HYBRID = 1, 2, 3
PATH_EXPECT_DT = np.dtype([("must", "<u4"), ("forbid", "<u4")])


@dataclass
class Workload:
    """A bag of numpy arrays plus the scalar sizes that go with them."""
    name: str
    seed: int
    arrays: dict = field(default_factory=dict)
    sizes: dict = field(default_factory=dict)
    meta: dict = field(default_factory=dict)

    def __getitem__(self, k):
        if k in self.arrays:
            return self.arrays[k]
        return self.sizes[k]

    def __contains__(self, k):
        return k in self.arrays or k in self.sizes


# ------------------------------------------------------------ primitives
def care_bits(rng, shape, p_care):
    """uint32 words whose bits are 1 with probability ~p_care, independently
    across bytes: each byte is drawn from the exact 8-bit product
    distribution quantised to 1/65536 (one 16-bit uniform draw per byte,
    inverse-CDF lookup).  The per-bit marginal is within 1e-4 of p_care."""
    if p_care <= 0:
        return np.zeros(shape, np.uint32)
    if p_care >= 1:
        return np.full(shape, 0xFFFFFFFF, np.uint32)
    lut = _byte_lut(float(p_care))
    n = int(np.prod(shape)) * 4
    u = rng.integers(0, 1 << 16, size=n, dtype=np.uint16)
    return lut[u].view(np.uint32).reshape(shape)


_LUTS: dict = {}


def _byte_lut(p):
    """65536-entry table: uniform 16-bit value -> byte with P(bit) = p."""
    if p not in _LUTS:
        b = np.arange(256)
        k = np.array([bin(x).count("1") for x in b])
        prob = p ** k * (1 - p) ** (8 - k)
        cdf = np.cumsum(prob)
        cdf /= cdf[-1]
        edges = np.round(cdf * 65536).astype(np.int64)
        lut = np.zeros(65536, np.uint8)
        lo = 0
        for x in range(256):
            hi = int(edges[x])
            lut[lo:hi] = x
            lo = hi
        _LUTS[p] = lut
    return _LUTS[p]


def distinct_values(rng, card, m, mmax=4):
    """For each row, `m` distinct values uniform over [0, card) (m <= card,
    m <= mmax).  Returns int32 [n, mmax] with -1 in unused slots."""
    card = np.asarray(card, np.int64)
    m = np.asarray(m, np.int64)
    n = card.shape[0]
    out = np.full((n, mmax), -1, np.int64)
    chosen = np.full((n, mmax), np.iinfo(np.int64).max, np.int64)  # sorted ascending
    for j in range(mmax):
        active = m > j
        hi = np.maximum(card - j, 1)
        r = rng.integers(0, hi)
        # map r to the r-th value not yet chosen (chosen kept sorted)
        for c in range(j):
            r = r + (r >= chosen[:, c])
        r = np.where(active, r, -1)
        out[:, j] = r
        # insert into sorted chosen
        ins = np.where(active, r, np.iinfo(np.int64).max)
        chosen[:, j] = ins
        chosen[:, : j + 1].sort(axis=1)
    return out.astype(np.int32)


def values_to_bitmap(vals):
    """int32 [n, k] values (-1 = unused) -> uint64 [n, 4] 256-bit set."""
    n = vals.shape[0]
    bm = np.zeros((n, 4), np.uint64)
    for j in range(vals.shape[1]):
        v = vals[:, j]
        ok = v >= 0
        w = np.where(ok, v >> 6, 0)
        b = np.where(ok, np.left_shift(np.uint64(1), (v & 63).astype(np.uint64)), np.uint64(0))
        np.bitwise_or.at(bm, (np.arange(n), w), b)
    return bm


# --------------------------------------------------------------- cluster
def gen_labels(rng, N, cards, absent_p=0.0):
    cards = np.asarray(cards, np.int64)
    L = cards.shape[0]
    labels = rng.integers(0, cards[None, :], size=(N, L)).astype(np.uint8)
    if absent_p > 0:
        labels[rng.random((N, L)) < absent_p] = ABSENT
    return labels


def gen_preds(rng, I, cards, kmin, kmax, mmax=4, op_p=None):
    """I selector rows, each a conjunction of k ~ U{kmin..kmax} predicates.
    Label uniform (with replacement), op uniform over In/NotIn/Exists
    (or op_p), In and NotIn value sets of m ~ U{1..mmax} distinct values
    clipped to the label's cardinality."""
    cards = np.asarray(cards, np.int64)
    L = cards.shape[0]
    k = rng.integers(kmin, kmax + 1, size=I)
    off = np.zeros(I + 1, np.int32)
    off[1:] = np.cumsum(k)
    P = int(off[-1])
    lab = rng.integers(0, L, size=P)
    if op_p is None:
        op = rng.integers(0, 3, size=P)
    else:
        op = rng.choice(3, size=P, p=op_p)
    card = cards[lab]
    m = np.minimum(rng.integers(1, mmax + 1, size=P), card)
    vals = distinct_values(rng, card, m, mmax)
    preds = np.zeros(P, PRED_DT)
    preds["label"] = lab
    preds["op"] = op
    bm = values_to_bitmap(vals)
    bm[op == OP_EXISTS] = 0
    preds["vals"] = bm
    return off, preds


def gen_affinity(rng, I, cards, tmin=1, tmax=3, kmin=1, kmax=4, mmax=4):
    """I required-affinity rows: t ~ U{tmin..tmax} terms per row, each a
    conjunction of k ~ U{kmin..kmax} expressions.  Label uniform, operator
    uniform over the six (In, NotIn, Exists, DoesNotExist, Gt, Lt); In and
    NotIn value sets as gen_preds; Gt and Lt thresholds uniform over
    [-1, card] (so some admit every value and some none), stored as a
    signed integer in vals[0].  Returns (row_off [I+1], term_off [T+1],
    preds)."""
    cards = np.asarray(cards, np.int64)
    L = cards.shape[0]
    t = rng.integers(tmin, tmax + 1, size=I)
    row_off = np.zeros(I + 1, np.int32)
    row_off[1:] = np.cumsum(t)
    T = int(row_off[-1])
    k = rng.integers(kmin, kmax + 1, size=T)
    term_off = np.zeros(T + 1, np.int32)
    term_off[1:] = np.cumsum(k)
    P = int(term_off[-1])
    lab = rng.integers(0, L, size=P)
    op = rng.integers(0, 6, size=P)
    card = cards[lab]
    m = np.minimum(rng.integers(1, mmax + 1, size=P), card)
    vals = distinct_values(rng, card, m, mmax)
    thr = rng.integers(-1, card + 1)
    preds = np.zeros(P, PRED_DT)
    preds["label"] = lab
    preds["op"] = op
    bm = values_to_bitmap(vals)
    setop = (op == OP_IN) | (op == OP_NOTIN)
    bm[~setop] = 0
    cmp = (op == OP_GT) | (op == OP_LT)
    bm[cmp, 0] = thr[cmp].astype(np.int64).view(np.uint64)
    preds["vals"] = bm
    return row_off, term_off, preds


def affinity_workload(seed, N, L, I, card_choices=(2, 4, 16, 64), absent_p=0.0, tmin=1, tmax=3, kmin=1, kmax=4,
                      name="affinity"):
    """N nodes x L uint8 labels (cardinality from card_choices, values
    uniform, a fraction absent_p absent) and I required-affinity rows
    (gen_affinity)."""
    rng = np.random.default_rng([seed, 11])
    cards = rng.choice(np.asarray(card_choices), size=L)
    labels = gen_labels(rng, N, cards, absent_p)
    row_off, term_off, preds = gen_affinity(rng, I, cards, tmin, tmax, kmin, kmax)
    wl = Workload(name, seed)
    wl.arrays.update(labels=labels, row_off=row_off, term_off=term_off, preds=preds)
    wl.sizes.update(N=N, L=L, I=I, n_terms=int(term_off.shape[0] - 1), n_preds=int(preds.shape[0]))
    wl.meta["cards"] = cards
    return wl


def affinity_rows(seed, cards, I, tmin=1, tmax=3, kmin=1, kmax=4):
    """I required-affinity rows (gen_affinity) over a cluster whose labels
    have the given cardinalities, from their own generator [seed, 12]."""
    return gen_affinity(np.random.default_rng([seed, 12]), I, cards, tmin, tmax, kmin, kmax)


def preferred_rows(seed, cards, I, tmin=1, tmax=3, kmin=1, kmax=3):
    """I preferred-affinity rows over a cluster whose labels have the given
    cardinalities, from their own generator [seed, 15]: terms and
    expressions as gen_affinity, and one weight per term, uniform over the
    Kubernetes range 1..100.  Returns (row_off, term_off, preds, weight)."""
    rng = np.random.default_rng([seed, 15])
    row_off, term_off, preds = gen_affinity(rng, I, cards, tmin, tmax, kmin, kmax)
    weight = rng.integers(1, 101, size=term_off.shape[0] - 1).astype(np.uint32)
    return row_off, term_off, preds, weight


def gen_preds_holding(rng, labels, cards, a, b, kmin, kmax, mmax=4):
    """Selector rows built so that nodes a[r] and b[r] satisfy row r: In sets
    contain both endpoints' values, NotIn sets avoid them (a NotIn with no
    value left to pick becomes Exists).  Labels must have no absent values."""
    cards = np.asarray(cards, np.int64)
    L = cards.shape[0]
    R = a.shape[0]
    k = rng.integers(kmin, kmax + 1, size=R)
    off = np.zeros(R + 1, np.int32)
    off[1:] = np.cumsum(k)
    P = int(off[-1])
    row = np.repeat(np.arange(R), k)
    lab = rng.integers(0, L, size=P)
    op = rng.integers(0, 3, size=P)
    card = cards[lab]
    va = labels[a[row], lab].astype(np.int64)
    vb = labels[b[row], lab].astype(np.int64)
    m = np.minimum(rng.integers(1, mmax + 1, size=P), card)
    cand = distinct_values(rng, card, np.minimum(card, mmax), mmax)
    one = np.uint64(1)

    def bit(v):
        return np.left_shift(one, (v & 63).astype(np.uint64)), (v >> 6)

    bm = np.zeros((P, 4), np.uint64)
    cnt = np.zeros(P, np.int64)
    isin = op == OP_IN
    # In: both endpoint values first
    for v in (va, vb):
        bv, w = bit(v)
        cur = bm[np.arange(P), w]
        new = isin & ((cur & bv) == 0)
        bm[np.arange(P)[new], w[new]] |= bv[new]
        cnt += new
    isnot = op == OP_NOTIN
    for j in range(mmax):
        c = cand[:, j].astype(np.int64)
        valid = c >= 0
        cc = np.where(valid, c, 0)
        bv, w = bit(cc)
        cur = bm[np.arange(P), w]
        fresh = valid & ((cur & bv) == 0) & (cnt < m)
        fresh &= isin | (isnot & (cc != va) & (cc != vb))
        fresh &= op != OP_EXISTS
        bm[np.arange(P)[fresh], w[fresh]] |= bv[fresh]
        cnt += fresh
    empty_notin = isnot & (cnt == 0)
    op = np.where(empty_notin, OP_EXISTS, op)
    bm[op == OP_EXISTS] = 0
    preds = np.zeros(P, PRED_DT)
    preds["label"] = lab
    preds["op"] = op
    preds["vals"] = bm
    return off, preds


# -------------------------------------------------------------- topology
def fat_tree(k, J):
    """k-ary fat-tree.  Pod p: edge e -> p*k+e, agg a -> p*k+k/2+a;
    core (i, j) -> k*k + i*k/2 + j.  Edge ports 0..k/2-1 face hosts,
    k/2+a faces agg a.  Agg ports 0..k/2-1 face edge e, k/2+j face core
    (a, j).  Core (i, j) port p faces agg i of pod p.  Jurisdiction of a
    pod switch is floor(p*J/k); core number c gets c mod J."""
    assert k % 2 == 0
    h = k // 2
    n_pod = k * k
    n_core = h * h
    S = n_pod + n_core
    nports = np.full(S, k, np.int32)
    port_off = np.zeros(S + 1, np.int32)
    port_off[1:] = np.cumsum(nports)
    peer = np.full(S * k, -1, np.int32)
    jur = np.zeros(S, np.uint8)
    for p in range(k):
        for e in range(h):
            s = p * k + e
            jur[s] = (p * J) // k
            for a in range(h):
                peer[port_off[s] + h + a] = p * k + h + a
        for a in range(h):
            s = p * k + h + a
            jur[s] = (p * J) // k
            for e in range(h):
                peer[port_off[s] + e] = p * k + e
            for j in range(h):
                peer[port_off[s] + h + j] = n_pod + a * h + j
    for i in range(h):
        for j in range(h):
            c = i * h + j
            s = n_pod + c
            jur[s] = c % J
            for p in range(k):
                peer[port_off[s] + p] = p * k + h + i
    H = k * k * k // 4
    hosts = np.arange(H)
    host_pod = hosts // (h * h)
    host_edge_local = (hosts // h) % h
    host_port = (hosts % h).astype(np.int32)
    host_switch = (host_pod * k + host_edge_local).astype(np.int32)
    host_ip = ((10 << 24) | (host_pod << 16) | (host_edge_local << 8) | (host_port + 2)).astype(np.uint32)
    topo = dict(kind="fat_tree", k=k, J=J, S=S, port_off=port_off, port_peer=peer, jur=jur,
                H=H, host_switch=host_switch, host_port=host_port, host_ip=host_ip)
    topo.update(_csr_from_ports(S, port_off, peer))
    return topo


def _csr_from_ports(S, port_off, peer):
    src = np.repeat(np.arange(S, dtype=np.int64), np.diff(port_off))
    m = peer >= 0
    u = src[m]
    v = peer[m].astype(np.int64)
    order = np.lexsort((v, u))
    u, v = u[order], v[order]
    adj_off = np.zeros(S + 1, np.int32)
    np.add.at(adj_off, u + 1, 1)
    adj_off = np.cumsum(adj_off).astype(np.int32)
    return dict(adj_off=adj_off, adj=v.astype(np.int32))


def random_graph(rng, S, E, hosts_per_switch, J):
    """Connected random graph: vertex i>0 attaches to a uniform earlier
    vertex (a random spanning tree), then uniform extra edges until |E|
    edges (no self-loops or duplicates).  Ports: link ports in neighbour-id
    order, then host ports.  Jurisdiction uniform over J."""
    parent = np.full(S, -1, np.int64)
    edges = set()
    for i in range(1, S):
        p = int(rng.integers(0, i))
        parent[i] = p
        edges.add((p, i))
    while len(edges) < E:
        u, v = (int(x) for x in rng.integers(0, S, size=2))
        if u == v:
            continue
        e = (min(u, v), max(u, v))
        edges.add(e)
    nbr = [[] for _ in range(S)]
    for u, v in sorted(edges):
        nbr[u].append(v)
        nbr[v].append(u)
    for l in nbr:
        l.sort()
    nports = np.array([len(nbr[s]) + hosts_per_switch for s in range(S)], np.int32)
    port_off = np.zeros(S + 1, np.int32)
    port_off[1:] = np.cumsum(nports)
    peer = np.full(int(port_off[-1]), -1, np.int32)
    for s in range(S):
        for i, v in enumerate(nbr[s]):
            peer[port_off[s] + i] = v
    jur = rng.integers(0, J, size=S).astype(np.uint8)
    H = S * hosts_per_switch
    hosts = np.arange(H)
    host_switch = (hosts // hosts_per_switch).astype(np.int32)
    host_port = np.array([len(nbr[s]) + (hh % hosts_per_switch) for hh, s in zip(hosts, host_switch)], np.int32)
    host_ip = ((10 << 24) | (host_switch.astype(np.int64) << 8) | (hosts % hosts_per_switch + 2)).astype(np.uint32)
    topo = dict(kind="random_graph", S=S, J=J, port_off=port_off, port_peer=peer, jur=jur,
                H=H, host_switch=host_switch, host_port=host_port, host_ip=host_ip,
                tree_parent=parent, nbr=nbr)
    topo.update(_csr_from_ports(S, port_off, peer))
    return topo


def _tree_path(parent, u, v):
    """Vertices on the spanning-tree path u -> v (parent pointers)."""
    anc_u = [u]
    while parent[anc_u[-1]] >= 0:
        anc_u.append(int(parent[anc_u[-1]]))
    pos = {x: i for i, x in enumerate(anc_u)}
    path_v = [v]
    while path_v[-1] not in pos:
        path_v.append(int(parent[path_v[-1]]))
    lca = path_v[-1]
    up = anc_u[: pos[lca] + 1]
    down = path_v[:-1][::-1]
    return up + down


def flow_paths(rng, topo, src_host, dst_host):
    """Per flow, the switches it crosses and the out-port used at each.
    Fat-tree: ECMP-style choice of a random aggregation and core switch.
    Random graph: the spanning-tree path.  Returns (sw [F,H], port [F,H], nh [F])."""
    F = src_host.shape[0]
    hs, hd = src_host.astype(np.int64), dst_host.astype(np.int64)
    if topo["kind"] == "fat_tree":
        k = topo["k"]
        h = k // 2
        n_pod = k * k
        Es = topo["host_switch"][hs].astype(np.int64)
        Ed = topo["host_switch"][hd].astype(np.int64)
        ps, pd = Es // k, Ed // k
        ed = Ed % k
        pdst = topo["host_port"][hd].astype(np.int64)
        a = rng.integers(0, h, size=F)
        j = rng.integers(0, h, size=F)
        sw = np.full((F, 5), -1, np.int64)
        port = np.full((F, 5), -1, np.int64)
        same_edge = Es == Ed
        same_pod = (ps == pd) & ~same_edge
        other = ps != pd
        # same edge
        sw[same_edge, 0] = Es[same_edge]
        port[same_edge, 0] = pdst[same_edge]
        # same pod: edge -> agg a -> edge
        m = same_pod
        sw[m, 0] = Es[m]; port[m, 0] = h + a[m]
        sw[m, 1] = ps[m] * k + h + a[m]; port[m, 1] = ed[m]
        sw[m, 2] = Ed[m]; port[m, 2] = pdst[m]
        # other pod: edge -> agg a -> core (a, j) -> agg a (dst pod) -> edge
        m = other
        sw[m, 0] = Es[m]; port[m, 0] = h + a[m]
        sw[m, 1] = ps[m] * k + h + a[m]; port[m, 1] = h + j[m]
        sw[m, 2] = n_pod + a[m] * h + j[m]; port[m, 2] = pd[m]
        sw[m, 3] = pd[m] * k + h + a[m]; port[m, 3] = ed[m]
        sw[m, 4] = Ed[m]; port[m, 4] = pdst[m]
        nh = np.where(same_edge, 1, np.where(same_pod, 3, 5))
        return sw, port, nh
    parent = topo["tree_parent"]
    nbr = topo["nbr"]
    paths = []
    for f in range(F):
        u = int(topo["host_switch"][hs[f]])
        v = int(topo["host_switch"][hd[f]])
        paths.append(_tree_path(parent, u, v))
    Hm = max(len(p) for p in paths) if paths else 1
    sw = np.full((F, Hm), -1, np.int64)
    port = np.full((F, Hm), -1, np.int64)
    nh = np.zeros(F, np.int64)
    for f, p in enumerate(paths):
        nh[f] = len(p)
        for i, s in enumerate(p):
            sw[f, i] = s
            if i + 1 < len(p):
                port[f, i] = nbr[s].index(p[i + 1])
            else:
                port[f, i] = topo["host_port"][hd[f]]
    return sw, port, nh


def flow_keys(rng, topo, src_host, dst_host):
    F = src_host.shape[0]
    keys = np.zeros((F, 4), np.uint32)
    keys[:, 0] = topo["host_ip"][src_host]
    keys[:, 1] = topo["host_ip"][dst_host]
    sport = rng.integers(0, 1 << 16, size=F, dtype=np.uint32)
    dport = rng.integers(0, 1 << 16, size=F, dtype=np.uint32)
    keys[:, 2] = (sport << np.uint32(16)) | dport
    keys[:, 3] = rng.integers(0, 256, size=F, dtype=np.uint32)
    return keys


def random_keys(rng, n):
    keys = rng.integers(0, 1 << 32, size=(n, 4), dtype=np.uint32)
    keys[:, 3] &= np.uint32(0xFF)
    return keys


def prefix_masks(rng, m, lo=16, hi=32):
    """Routing-table masks: a destination-address prefix of a uniform length
    in [lo, hi] bits; source address, ports and protocol wildcarded."""
    L = rng.integers(lo, hi + 1, size=m).astype(np.uint64)
    msk = np.zeros((m, 4), np.uint32)
    msk[:, 1] = ((np.uint64(0xFFFFFFFF) << (np.uint64(32) - L)) & np.uint64(0xFFFFFFFF)).astype(np.uint32)
    return msk


def build_tables(rng, topo, R, p_care, drop_p=0.05, misroute_p=0.02,
                 prio="distinct", prio_range=8, flows=None, chunk=256, masks="iid"):
    """R rules per switch.  Every slot first holds an i.i.d. rule (random
    value, care bits with probability p_care, action = uniform port or DROP
    with probability drop_p); then, when `flows` = (keys, sw, port, nh) is
    given, one rule per hop of every flow replaces a random free slot of
    that switch: value = flow key, action = the path's next port, except
    DROP with probability drop_p and a uniform port with probability
    misroute_p.  Priorities: 'distinct' (R distinct uint16 per switch in
    random order: a random permutation of R strata of width 65536/R, a
    uniform offset inside each), 'uniform' (i.i.d. uint16, ties possible) or
    'small' (uniform over [0, prio_range), many ties).  masks='prefix':
    every rule matches a destination prefix only (prefix_masks) instead of
    i.i.d. care bits."""
    S = topo["S"]
    mk = (lambda m: prefix_masks(rng, m)) if masks == "prefix" else None
    port_off = topo["port_off"]
    nports = np.diff(port_off).astype(np.int64)
    n = S * R
    assert n < 2**31
    rules = np.zeros(n, RULE_DT)
    raw = rules.view(np.uint32).reshape(n, 10)   # value[4], mask[4], prio | action << 16, rsv
    rule_off = (np.arange(S + 1, dtype=np.int64) * R).astype(np.int32)
    for s0 in range(0, S, chunk):
        s1 = min(S, s0 + chunk)
        m = (s1 - s0) * R
        val = random_keys(rng, m)
        msk = care_bits(rng, (m, 4), p_care) if mk is None else mk(m)
        msk[:, 3] &= np.uint32(0xFF)
        blk = np.empty((m, 10), np.uint32)
        blk[:, 0:4] = val & msk
        blk[:, 4:8] = msk
        np_ = np.repeat(nports[s0:s1], R)
        act = rng.integers(0, np.maximum(np_, 1))
        act = np.where(rng.random(m) < drop_p, DROP, act).astype(np.uint32)
        if prio == "distinct":
            assert R <= 65536
            width = 65536 // R
            strata = np.argsort(rng.random((s1 - s0, R)), axis=1).reshape(-1).astype(np.int64)
            pr = strata * width + rng.integers(0, width, size=m)
        elif prio == "uniform":
            pr = rng.integers(0, 65536, size=m)
        else:
            pr = rng.integers(0, prio_range, size=m)
        blk[:, 8] = pr.astype(np.uint32) | (act << np.uint32(16))
        blk[:, 9] = 0
        raw[s0 * R:s1 * R] = blk
    dropped = 0
    if flows is not None:
        keys, sw, port, nh = flows
        F, Hm = sw.shape
        hop = np.arange(Hm)[None, :] < nh[:, None]
        fidx = np.nonzero(hop)
        e_flow = fidx[0]
        e_sw = sw[fidx]
        e_port = port[fidx]
        ne = e_flow.shape[0]
        order = np.argsort(e_sw, kind="stable")
        e_flow, e_sw, e_port = e_flow[order], e_sw[order], e_port[order]
        cnt = np.bincount(e_sw, minlength=S)
        start = np.zeros(S + 1, np.int64)
        start[1:] = np.cumsum(cnt)
        rank = np.arange(ne) - start[e_sw]
        keep = rank < R
        dropped = int((~keep).sum())
        e_flow, e_sw, e_port, rank = e_flow[keep], e_sw[keep], e_port[keep], rank[keep]
        # slot = rank-th entry of a random permutation of the switch's R slots
        slot = np.empty(e_sw.shape[0], np.int64)
        for s0 in range(0, S, chunk):
            s1 = min(S, s0 + chunk)
            sel = (e_sw >= s0) & (e_sw < s1)
            if not sel.any():
                continue
            perm = np.argsort(rng.random((s1 - s0, R)), axis=1)
            slot[sel] = perm[e_sw[sel] - s0, rank[sel]]
        pos = e_sw * R + slot
        m = pos.shape[0]
        msk = care_bits(rng, (m, 4), p_care) if mk is None else mk(m)
        msk[:, 3] &= np.uint32(0xFF)
        raw[pos, 0:4] = keys[e_flow] & msk
        raw[pos, 4:8] = msk
        u = rng.random(m)
        mis = rng.integers(0, np.maximum(nports[e_sw], 1))
        act = np.where(u < drop_p, DROP, np.where(u < drop_p + misroute_p, mis, e_port)).astype(np.uint32)
        raw[pos, 8] = (raw[pos, 8] & np.uint32(0xFFFF)) | (act << np.uint32(16))
    return rule_off, rules, dropped


# ------------------------------------------------------------- workloads
def _selector_arrays(wl, labels, off, preds):
    wl.arrays.update(labels=labels, pred_off=off, preds=preds)
    wl.sizes.update(N=labels.shape[0], L=labels.shape[1], I_rows=off.shape[0] - 1,
                    n_preds=int(preds.shape[0]))


def _topo_arrays(wl, topo):
    wl.arrays.update(port_off=topo["port_off"], port_peer=topo["port_peer"], jur=topo["jur"],
                     adj_off=topo["adj_off"], adj=topo["adj"], region=topo["jur"].copy())
    wl.sizes.update(S=topo["S"], n_ports=int(topo["port_peer"].shape[0]), V=topo["S"],
                    n_adj=int(topo["adj"].shape[0]))


def selector_workload(seed, N, L, I, card_choices=(2, 4, 16, 64), kmin=1, kmax=8,
                      absent_p=0.0, name="selector"):
    """Selector evaluation only: N nodes x L uint8 labels with per-label
    cardinality drawn from card_choices and uniform values; I rows of
    kmin..kmax predicates."""
    rng = np.random.default_rng(seed)
    cards = rng.choice(np.asarray(card_choices), size=L)
    labels = gen_labels(rng, N, cards, absent_p)
    off, preds = gen_preds(rng, I, cards, kmin, kmax)
    wl = Workload(name, seed)
    _selector_arrays(wl, labels, off, preds)
    wl.meta["cards"] = cards
    return wl


def cfg2(seed=1):
    """100,000 nodes x 64 labels, cardinality from {2,4,16,64}; 16,384 rows
    of 1..8 predicates."""
    return selector_workload(seed, 100_000, 64, 16_384, name="cfg2")


def mutate_tables(seed, port_off, rule_off, rules, switches, resize=False):
    """New flow tables in which the listed switches' rules are rewritten:
    every rule of such a switch gets a fresh priority (a permutation of the
    old ones) and a fresh action (a random local port, DROP with probability
    0.1).  resize=True also drops the last rule of every other listed switch
    and repeats the first rule of the rest, so table sizes change too.
    Other switches keep their rules.  Returns (rule_off, rules)."""
    rng = np.random.default_rng([seed, 16])
    rule_off = np.asarray(rule_off, np.int64)
    S = rule_off.shape[0] - 1
    chosen = set(int(x) for x in switches if 0 <= int(x) < S)
    parts = []
    for s_ in range(S):
        seg = rules[rule_off[s_]:rule_off[s_ + 1]].copy()
        if s_ in chosen and seg.shape[0] > 0:
            seg["priority"] = rng.permutation(seg["priority"])
            npt = int(port_off[s_ + 1] - port_off[s_])
            act = rng.integers(0, max(npt, 1), size=seg.shape[0]).astype(np.uint16)
            act[rng.random(seg.shape[0]) < 0.1] = 0xFFFF
            seg["action"] = act
            if resize:
                seg = seg[:-1] if s_ % 2 == 0 else np.concatenate([seg, seg[:1]])
        parts.append(seg)
    new_off = np.zeros(S + 1, np.int32)
    new_off[1:] = np.cumsum([p.shape[0] for p in parts])
    new_rules = np.concatenate(parts) if parts else rules[:0].copy()
    return new_off, new_rules


def trace_workload(seed, k, J, R, T, ttl, n_flows, p_care=0.7, variant="rpath",
                   name="trace"):
    """Flow tracing only on a k-ary fat-tree with J jurisdictions by pod and
    R rules per switch.  variant 'rpath': n_flows flows between random host
    pairs, each compiled into one rule per hop; T headers drawn uniformly
    from the flows and injected at the flow's ingress edge switch.
    'literal': i.i.d. rules only and uniform random headers at random edge
    switches.  'dense': 95% wildcard bits, small priority range, i.i.d.
    rules, random headers at random switches.  'prefix': as 'rpath', but
    every rule (path or noise) matches a destination prefix of 16-32 bits
    with ports, source and protocol wildcarded, as a routing table does."""
    rng = np.random.default_rng(seed)
    topo = fat_tree(k, J)
    wl = Workload(name, seed)
    wl.meta.update(variant=variant, k=k, J=J, R=R)
    if variant in ("rpath", "prefix"):
        H = topo["H"]
        hs = rng.integers(0, H, size=n_flows)
        hd = (hs + rng.integers(1, H, size=n_flows)) % H
        keys = flow_keys(rng, topo, hs, hd)
        sw, port, nh = flow_paths(rng, topo, hs, hd)
        rule_off, rules, dropped = build_tables(rng, topo, R, p_care, flows=(keys, sw, port, nh),
                                                masks="iid" if variant == "rpath" else "prefix")
        pick = rng.integers(0, n_flows, size=T)
        hdr = keys[pick]
        ingress = topo["host_switch"][hs[pick]].astype(np.int32)
        wl.meta["path_rules_dropped"] = dropped
    elif variant == "literal":
        rule_off, rules, _ = build_tables(rng, topo, R, p_care)
        hdr = random_keys(rng, T)
        h = k // 2
        pods = rng.integers(0, k, size=T)
        ingress = (pods * k + rng.integers(0, h, size=T)).astype(np.int32)
    elif variant == "dense":
        rule_off, rules, _ = build_tables(rng, topo, R, 0.05, prio="small")
        hdr = random_keys(rng, T)
        ingress = rng.integers(0, topo["S"], size=T).astype(np.int32)
    else:
        raise ValueError(variant)
    _topo_arrays(wl, topo)
    wl.arrays.update(rule_off=rule_off, rules=rules, hdr=hdr, ingress=ingress)
    wl.sizes.update(T=T, ttl=ttl, n_rules=int(rules.shape[0]))
    return wl


def cfg3(seed=2, variant="rpath"):
    """Fat-tree k=32 (1,280 switches), 4,096 rules per switch, 30% wildcard
    bits, distinct priorities, 5% drop; 8 jurisdictions by pod; 4,194,304
    headers, TTL 32; 524,288 compiled flows."""
    return trace_workload(seed, 32, 8, 4096, 4_194_304, 32, 524_288, variant=variant, name="cfg3")


def rgg_workload(seed, V, n_regions, Q, mean_degree=4.0, full_rows=True, name="reach"):
    """Random geometric graph: V points uniform in the unit square, an edge
    when the Euclidean distance is below r = sqrt(mean_degree/(pi V)).
    Regions: Voronoi cells of n_regions uniform seeds (ties to the lower
    seed).  Queries allow k ~ U{1..8} distinct regions and start at a
    uniform vertex of an allowed region."""
    from scipy.spatial import cKDTree
    rng = np.random.default_rng(seed)
    pts = rng.random((V, 2))
    r = math.sqrt(mean_degree / (math.pi * V))
    pairs = cKDTree(pts).query_pairs(r, output_type="ndarray")
    if pairs.shape[0]:
        d2 = ((pts[pairs[:, 0]] - pts[pairs[:, 1]]) ** 2).sum(1)
        pairs = pairs[d2 < r * r]
    u = np.concatenate([pairs[:, 0], pairs[:, 1]]).astype(np.int64)
    v = np.concatenate([pairs[:, 1], pairs[:, 0]]).astype(np.int64)
    order = np.lexsort((v, u))
    u, v = u[order], v[order]
    adj_off = np.zeros(V + 1, np.int64)
    np.add.at(adj_off, u + 1, 1)
    adj_off = np.cumsum(adj_off).astype(np.int32)
    seeds = rng.random((n_regions, 2))
    region = np.empty(V, np.uint8)
    for c0 in range(0, V, 1 << 18):
        c1 = min(V, c0 + (1 << 18))
        d = ((pts[c0:c1, None, :] - seeds[None, :, :]) ** 2).sum(2)
        region[c0:c1] = np.argmin(d, axis=1)
    allowed = np.zeros(Q, np.uint32)
    src = np.zeros(Q, np.int32)
    for q in range(Q):
        kq = int(rng.integers(1, min(8, n_regions) + 1))
        regs = rng.choice(n_regions, size=kq, replace=False)
        allowed[q] = np.bitwise_or.reduce(np.left_shift(np.uint32(1), regs.astype(np.uint32)))
        cand = np.flatnonzero(np.isin(region, regs))
        src[q] = cand[rng.integers(0, cand.shape[0])]
    wl = Workload(name, seed)
    wl.arrays.update(adj_off=adj_off, adj=v.astype(np.int32), region=region, src=src,
                     allowed=allowed, pts=pts)
    if not full_rows:
        wl.arrays["target"] = rng.integers(0, V, size=Q).astype(np.int32)
    wl.sizes.update(V=V, n_adj=int(v.shape[0]), Q=Q)
    wl.meta.update(radius=r)
    return wl


def cfg4(seed=3):
    """Random geometric graph of 1,000,000 switches, mean degree 4,
    16-region Voronoi map, 256 queries, full distance rows."""
    return rgg_workload(seed, 1_000_000, 16, 256, name="cfg4")


def path_constraints(seed, S, sw, nh, n_forbid=2, p_on_path=0.5, p_forbid_on_path=0.125):
    """Required waypoint and forbidden switches per flow (the routing
    constraints of a Configuration: must-go waypoints and forbidden
    vertices).  Flow f's compiled path is sw[f, :nh[f]].  The waypoint is,
    with probability p_on_path, a uniform interior switch of the path (its
    only switch when it has no interior), else a uniform switch.  Each of
    the n_forbid forbidden switches is, with probability p_forbid_on_path, an
    interior switch of the path, else a uniform switch; none equals the
    waypoint.  Uses its own generator (seed, 7), so the other arrays of a
    workload do not change.  Returns (via [F, 1], forbid [F, n_forbid])."""
    rng = np.random.default_rng([seed, 7])
    F = sw.shape[0]
    nh = np.asarray(nh, np.int64)
    n_in = np.maximum(nh - 2, 0)

    def pick_interior():
        j = np.where(n_in > 0, 1 + (rng.random(F) * np.maximum(n_in, 1)).astype(np.int64), 0)
        return sw[np.arange(F), j].astype(np.int64)

    way = np.where(rng.random(F) < p_on_path, pick_interior(), rng.integers(0, S, size=F))
    forbid = np.empty((F, n_forbid), np.int64)
    for c in range(n_forbid):
        f = np.where(rng.random(F) < p_forbid_on_path, pick_interior(), rng.integers(0, S, size=F))
        for _ in range(64):
            bad = f == way
            if not bad.any():
                break
            f[bad] = rng.integers(0, S, size=int(bad.sum()))
        f[f == way] = -1
        forbid[:, c] = f
    return way[:, None].astype(np.int32), forbid.astype(np.int32)


def port_weights(seed, n_ports, wmax=10):
    """Link weights per port, uniform over 1..wmax, from their own
    generator [seed, 13] (latency-like costs for a weighted path search)."""
    return np.random.default_rng([seed, 13]).integers(1, wmax + 1, size=n_ports).astype(np.uint32)


def synthesis_requests(seed, topo, Q, Kv=1, Kf=2, p_via=0.7, p_other_jur=0.5):
    """Q path-synthesis requests between uniform distinct hosts of a
    topology: source and target are the hosts' switches, out_port the
    destination host's port, key a fresh random 5-tuple per request.  The
    allowed jurisdictions are both endpoints' plus each other one with
    probability p_other_jur; up to Kv waypoints (as many as slots drawn
    with probability p_via, in the first slots; uniform switches; the list
    ends at its first -1) and Kf uniform forbidden switches
    (-1 when one would hit an endpoint or a waypoint).  Own generator
    [seed, 14]."""
    rng = np.random.default_rng([seed, 14])
    S, J, H = topo["S"], topo["J"], topo["H"]
    a = rng.integers(0, H, size=Q)
    b = (a + rng.integers(1, H, size=Q)) % H
    src = topo["host_switch"][a].astype(np.int32)
    dst = topo["host_switch"][b].astype(np.int32)
    out_port = topo["host_port"][b].astype(np.int32)
    jur = topo["jur"].astype(np.int64)
    allowed = (np.left_shift(1, jur[src]) | np.left_shift(1, jur[dst])).astype(np.uint32)
    for j in range(J):
        allowed |= np.where(rng.random(Q) < p_other_jur, np.uint32(1 << j), np.uint32(0))
    # waypoint lists end at their first -1 (used slots first)
    n_via = (rng.random((Q, Kv)) < p_via).sum(axis=1)
    via = np.where(np.arange(Kv)[None, :] < n_via[:, None], rng.integers(0, S, size=(Q, Kv)), -1).astype(np.int32)
    forbid = rng.integers(0, S, size=(Q, Kf)).astype(np.int32)
    clash = (forbid == src[:, None]) | (forbid == dst[:, None])
    for c in range(Kv):
        clash |= forbid == via[:, c:c + 1]
    forbid[clash] = -1
    key = random_keys(rng, Q)
    return dict(src=src, target=dst, out_port=out_port, allowed=allowed, via=via, forbid=forbid, key=key)


def _add_paths(wl, via_q, forb_q, trace_q, pexp_rows):
    """Attach path constraints: query q's via / forbid lists; trace t
    watches [waypoint, forbidden...] of its query trace_q[t]; network
    intents expect the waypoint in slot 0 and the rest forbidden."""
    watch = np.concatenate([via_q, forb_q], axis=1)[trace_q]
    K = watch.shape[1]
    pexp = np.zeros(wl["intents"].shape[0], PATH_EXPECT_DT)
    pexp["must"][pexp_rows] = 1
    pexp["forbid"][pexp_rows] = ((1 << K) - 1) & ~1
    wl.arrays.update(via=via_q, forbid=forb_q, watch=np.ascontiguousarray(watch, np.int32), pexp=pexp)


def combined_workload(seed, N, L, k, J, R, I, ttl=32, p_care=0.7, kmin=1, kmax=8,
                      card_choices=(2, 4, 16, 64), name="combined", paths=False):
    """Cross-layer validation: kind = [compute, network, hybrid][i mod 3].
    Compute and hybrid intents own a selector row (1..kmax predicates).
    Network intents join two distinct uniform hosts; hybrid intents join
    the hosts of two distinct nodes (node n sits on host n mod H) whose
    selector row is built to hold for both, except that 1 in 16 have their
    destination placed on a uniform node instead (which the row may not
    admit).  Every network and hybrid
    intent owns one flow (compiled one rule per hop into the tables), one
    trace of the flow's header from its ingress edge switch, and one
    reachability query from the ingress to the egress edge switch.  The
    allowed jurisdictions are those of both edge switches plus each other
    jurisdiction with probability 1/2.  paths=True adds a waypoint and two
    forbidden switches per flow (path_constraints)."""
    rng = np.random.default_rng(seed)
    cards = rng.choice(np.asarray(card_choices), size=L)
    labels = gen_labels(rng, N, cards)
    topo = fat_tree(k, J)
    H = topo["H"]
    kind = np.array([KIND_COMPUTE, KIND_NETWORK, KIND_HYBRID], np.uint8)[np.arange(I) % 3]
    has_sel = (kind & 1) == 1
    has_net = (kind & 2) == 2
    sel_row = np.full(I, -1, np.int32)
    sel_row[has_sel] = np.arange(int(has_sel.sum()), dtype=np.int32)
    comp_idx = np.flatnonzero(kind == KIND_COMPUTE)
    hyb_idx = np.flatnonzero(kind == KIND_HYBRID)
    net_idx = np.flatnonzero(kind == KIND_NETWORK)
    # hybrid endpoints: distinct nodes on distinct hosts
    a = rng.integers(0, N, size=hyb_idx.shape[0])
    b = rng.integers(0, N, size=hyb_idx.shape[0])
    for _ in range(64):
        bad = (a == b) | (a % H == b % H)
        if not bad.any():
            break
        b[bad] = rng.integers(0, N, size=int(bad.sum()))
    # selector rows, in sel_row order
    off_c, preds_c = gen_preds(rng, comp_idx.shape[0], cards, kmin, kmax)
    off_h, preds_h = gen_preds_holding(rng, labels, cards, a, b, kmin, kmax)
    # a misplaced deployment: 1 in 16 hybrid intents have their destination
    # pod placed on a uniform node instead (own stream, so nothing else moves);
    # the row was built for the intended node, so the placed one may fail it
    rng_m = np.random.default_rng([seed, 9])
    mis = rng_m.random(hyb_idx.shape[0]) < 1.0 / 16
    b_m = rng_m.integers(0, N, size=hyb_idx.shape[0])
    ok_m = (b_m != a) & (b_m % H != a % H)
    b = np.where(mis & ok_m, b_m, b)
    rows = int(has_sel.sum())
    k_row = np.zeros(rows, np.int64)
    k_row[sel_row[comp_idx]] = np.diff(off_c)
    k_row[sel_row[hyb_idx]] = np.diff(off_h)
    pred_off = np.zeros(rows + 1, np.int64)
    pred_off[1:] = np.cumsum(k_row)
    preds = np.zeros(int(pred_off[-1]), PRED_DT)
    for idx, off, pr in ((comp_idx, off_c, preds_c), (hyb_idx, off_h, preds_h)):
        r = sel_row[idx]
        cnt = np.diff(off)
        dst = np.repeat(pred_off[r], cnt) + (np.arange(int(cnt.sum())) - np.repeat(off[:-1], cnt))
        preds[dst] = pr
    pred_off = pred_off.astype(np.int32)
    # flows: one per network / hybrid intent, in intent order
    fl_int = np.flatnonzero(has_net)
    F = fl_int.shape[0]
    hs = np.empty(F, np.int64)
    hd = np.empty(F, np.int64)
    is_h = kind[fl_int] == KIND_HYBRID
    hs[is_h] = a % H
    hd[is_h] = b % H
    nn = int((~is_h).sum())
    s_ = rng.integers(0, H, size=nn)
    hs[~is_h] = s_
    hd[~is_h] = (s_ + rng.integers(1, H, size=nn)) % H
    keys = flow_keys(rng, topo, hs, hd)
    sw, port, nh = flow_paths(rng, topo, hs, hd)
    rule_off, rules, dropped = build_tables(rng, topo, R, p_care, flows=(keys, sw, port, nh))
    e_src = topo["host_switch"][hs].astype(np.int32)
    e_dst = topo["host_switch"][hd].astype(np.int32)
    jur = topo["jur"].astype(np.int64)
    allowed = (np.left_shift(1, jur[e_src]) | np.left_shift(1, jur[e_dst])).astype(np.uint32)
    extra = rng.random((F, J)) < 0.5
    for j in range(J):
        allowed |= np.where(extra[:, j], np.uint32(1 << j), np.uint32(0))
    intents = np.zeros(I, INTENT_DT)
    intents["kind"] = kind
    intents["sel_row"] = sel_row
    intents["src_node"] = -1
    intents["dst_node"] = -1
    intents["src_node"][hyb_idx] = a
    intents["dst_node"][hyb_idx] = b
    intents["trace_begin"] = 0
    intents["trace_end"] = 0
    intents["trace_begin"][fl_int] = np.arange(F)
    intents["trace_end"][fl_int] = np.arange(F) + 1
    intents["allowed"][fl_int] = allowed
    expect = np.zeros(I, EXPECT_DT)
    expect["dst_switch"] = -1
    expect["dst_port"] = -1
    expect["reach_q"] = -1
    expect["dst_switch"][fl_int] = e_dst
    expect["dst_port"][fl_int] = topo["host_port"][hd]
    expect["reach_q"][fl_int] = np.arange(F)
    wl = Workload(name, seed)
    _selector_arrays(wl, labels, pred_off, preds)
    _topo_arrays(wl, topo)
    wl.arrays.update(rule_off=rule_off, rules=rules, hdr=keys, ingress=e_src,
                     src=e_src.copy(), allowed=allowed, target=e_dst.copy(),
                     intents=intents, expect=expect)
    wl.sizes.update(T=F, ttl=ttl, n_rules=int(rules.shape[0]), Q=F, I=I)
    wl.meta.update(k=k, J=J, R=R, cards=cards, path_rules_dropped=dropped)
    if paths:
        via, forb = path_constraints(seed, topo["S"], sw, nh)
        _add_paths(wl, via, forb, np.arange(F), fl_int)
    return wl


def cfg5(seed=4, paths=False):
    """50,000 nodes x 64 labels; fat-tree k=48 (2,880 switches), 16,384 rules
    per switch, 12 jurisdictions; 1,048,576 intents split evenly between
    compute-only, network-only and hybrid.  paths=True adds waypoint and
    forbidden-switch constraints."""
    return combined_workload(seed, 50_000, 64, 48, 12, 16_384, 1_048_576, name="cfg5", paths=paths)


def cfg1(seed=0, variant="rpath", paths=False):
    """Tiny end-to-end case: 16 nodes x 8 labels (region over 4, trust tier
    0..3, six categorical labels of cardinality 8); 12 switches on a random
    connected graph with 18 links (mean degree 3), 2 host ports each,
    jurisdiction over 4; 32 rules per switch with 50% wildcard bits and
    i.i.d. uint16 priorities; 64 intents of 1..3 predicates and a non-empty
    allowed subset; 1,024 traces with TTL 16.  variant 'rpath' compiles one
    flow per network/hybrid intent along the spanning-tree path; 'literal'
    uses i.i.d. rules and uniform headers at random switches; 'dense' uses
    95% wildcard bits and priorities in [0, 8).  paths=True adds a waypoint
    and two forbidden switches per network intent (path_constraints)."""
    rng = np.random.default_rng(seed)
    N, L, S, I, T, R, J, TTL = 16, 8, 12, 64, 1024, 32, 4, 16
    cards = np.array([4, 4, 8, 8, 8, 8, 8, 8], np.int64)
    labels = gen_labels(rng, N, cards)
    topo = random_graph(rng, S, 18, 2, J)
    H = topo["H"]
    kind = np.array([KIND_COMPUTE, KIND_NETWORK, KIND_HYBRID], np.uint8)[np.arange(I) % 3]
    has_sel = (kind & 1) == 1
    has_net = (kind & 2) == 2
    rows = int(has_sel.sum())
    sel_row = np.full(I, -1, np.int32)
    sel_row[has_sel] = np.arange(rows, dtype=np.int32)
    pred_off, preds = gen_preds(rng, rows, cards, 1, 3)
    src_node = np.full(I, -1, np.int32)
    dst_node = np.full(I, -1, np.int32)
    hyb = np.flatnonzero(kind == KIND_HYBRID)
    src_node[hyb] = rng.integers(0, N, size=hyb.shape[0])
    dst_node[hyb] = (src_node[hyb] + rng.integers(1, N, size=hyb.shape[0])) % N
    net = np.flatnonzero(has_net)
    nf = 1
    hs_i = np.empty(net.shape[0], np.int64)
    hd_i = np.empty(net.shape[0], np.int64)
    for j, i in enumerate(net):
        if kind[i] == KIND_HYBRID:
            hs_i[j], hd_i[j] = src_node[i] % H, dst_node[i] % H
        else:
            s_ = int(rng.integers(0, H))
            hs_i[j], hd_i[j] = s_, (s_ + int(rng.integers(1, H))) % H
    allowed = np.zeros(I, np.uint32)
    allowed[net] = rng.integers(1, 1 << J, size=net.shape[0]).astype(np.uint32)
    hs = np.repeat(hs_i, nf)
    hd = np.repeat(hd_i, nf)
    keys = flow_keys(rng, topo, hs, hd)
    sw, port, nh = flow_paths(rng, topo, hs, hd)
    # traces: contiguous ranges per network/hybrid intent
    per = np.full(net.shape[0], T // net.shape[0])
    per[: T - per.sum()] += 1
    tb = np.zeros(net.shape[0] + 1, np.int64)
    tb[1:] = np.cumsum(per)
    owner = np.repeat(np.arange(net.shape[0]), per)
    fl = owner * nf + rng.integers(0, nf, size=T)
    if variant == "rpath":
        rule_off, rules, dropped = build_tables(rng, topo, R, 0.5, prio="uniform",
                                                flows=(keys, sw, port, nh))
        hdr = keys[fl]
        ingress = topo["host_switch"][hs[fl]].astype(np.int32)
    elif variant == "literal":
        rule_off, rules, dropped = build_tables(rng, topo, R, 0.5, prio="uniform")
        hdr = random_keys(rng, T)
        ingress = rng.integers(0, S, size=T).astype(np.int32)
    elif variant == "dense":
        rule_off, rules, dropped = build_tables(rng, topo, R, 0.05, prio="small")
        hdr = random_keys(rng, T)
        ingress = rng.integers(0, S, size=T).astype(np.int32)
    else:
        raise ValueError(variant)
    intents = np.zeros(I, INTENT_DT)
    intents["kind"] = kind
    intents["sel_row"] = sel_row
    intents["src_node"] = src_node
    intents["dst_node"] = dst_node
    intents["trace_begin"][net] = tb[:-1]
    intents["trace_end"][net] = tb[1:]
    intents["allowed"] = allowed
    expect = np.zeros(I, EXPECT_DT)
    expect["dst_switch"] = -1
    expect["dst_port"] = -1
    expect["reach_q"] = -1
    expect["dst_switch"][net] = topo["host_switch"][hd_i]
    expect["dst_port"][net] = topo["host_port"][hd_i]
    expect["reach_q"][net] = np.arange(net.shape[0])
    wl = Workload("cfg1", seed)
    _selector_arrays(wl, labels, pred_off, preds)
    _topo_arrays(wl, topo)
    wl.arrays.update(rule_off=rule_off, rules=rules, hdr=hdr, ingress=ingress,
                     src=topo["host_switch"][hs_i].astype(np.int32), allowed=allowed[net].copy(),
                     target=topo["host_switch"][hd_i].astype(np.int32),
                     intents=intents, expect=expect)
    wl.sizes.update(T=T, ttl=TTL, n_rules=int(rules.shape[0]), Q=int(net.shape[0]), I=I)
    wl.meta.update(variant=variant, cards=cards, path_rules_dropped=dropped, topo=topo)
    if paths:
        via, forb = path_constraints(seed, S, sw, nh)
        _add_paths(wl, via, forb, owner, net)
    return wl


CONFIGS = {"cfg1": cfg1, "cfg2": cfg2, "cfg3": cfg3, "cfg4": cfg4, "cfg5": cfg5}
