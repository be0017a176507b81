"""Parity of pc_trace_flows_delta (through the C ABI) with the CPU oracle:
after the rules of some switches change, re-tracing only the traces whose
visited-switch summary meets a changed switch gives exactly the oracle's
full trace on the new tables (records and summaries, bit-exact), starting
from the oracle's old results or from the GPU's own, over chains of
changes, with resized tables, repeated and out-of-range ids, no change,
every switch changed and no traces; and at the combined workload's size."""
import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu
F_SWITCH = 8


@pytest.fixture(scope="module")
def g():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import gpu_run
    return gpu_run


def _run(wl, rule_off, rules, out, vsum, changed, walk=None, use_walk=True, ctx=None):
    """One delta call; out / vsum / walk as numpy (records, u64, int32
    [T, 8]) or None for a first call.  Returns (records, vsum, walk,
    n_retraced, flags); walk is None with use_walk=False.  Without ctx a
    fresh context (no prepared tables kept) serves the call; a chain of calls
    on the same tables passes its own context."""
    import torch
    import paper_2602_16100_amd as pc
    ctx = ctx or pc.Context(0)
    ctx.data_errors(clear=True)
    T = wl["ingress"].shape[0]
    d = lambda a: pc.to_device(a, "cuda")
    o = torch.zeros((T, 12), dtype=torch.uint8, device="cuda") if out is None else \
        torch.from_numpy(np.ascontiguousarray(out).view(np.uint8).reshape(T, 12).copy()).cuda()
    v = torch.zeros(T, dtype=torch.int64, device="cuda") if vsum is None else \
        torch.from_numpy(np.ascontiguousarray(vsum, np.uint64).view(np.int64).copy()).cuda()
    ch = None if changed is None else torch.from_numpy(np.ascontiguousarray(changed, np.int32)).cuda()
    w = None
    if use_walk:
        w = torch.full((T, 8), -5, dtype=torch.int32, device="cuda") if walk is None else \
            torch.from_numpy(np.ascontiguousarray(walk, np.int32).copy()).cuda()
    n = pc.pc_trace_flows_delta(wl["S"], d(wl["port_off"]), d(wl["port_peer"]), d(wl["jur"]), d(rule_off), d(rules),
                                d(np.ascontiguousarray(wl["hdr"], np.uint32)), d(wl["ingress"]), wl["ttl"], o, v,
                                changed=ch, walk=w, ctx=ctx)
    torch.cuda.synchronize()
    flags = ctx.data_errors(clear=True)
    return (pc.records(o, pc.TRACE_OUT_DT), v.cpu().numpy().view(np.uint64),
            None if w is None else w.cpu().numpy(), int(n.cpu().numpy()[0]), flags)


def _oracle(orc, wl, rule_off, rules, idx=None):
    return orc.trace(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], rule_off, rules, wl["hdr"], wl["ingress"],
                     wl["ttl"], idx=idx, summary=True)


def _same_records(a, b):
    for f in ("jmask", "last_switch", "last_port", "hops", "state"):
        bad = np.flatnonzero(a[f] != b[f])
        assert bad.size == 0, f"{f}: first mismatch at trace {bad[0]}: gpu {a[bad[0]]} oracle {b[bad[0]]}"


def _mask(changed):
    m = 0
    for s in changed:
        m |= 1 << (int(s) & 63)
    return np.uint64(m)


def _expected_count(ro, vo, wo, changed, use_walk=True):
    """Traces to trace again: exact for walks that fit their record, by
    summary bits otherwise (or always, without records)."""
    by_sum = (vo & _mask(changed)) != 0
    if not use_walk:
        return int(by_sum.sum())
    ch = np.asarray([c for c in changed if c >= 0], np.int64)
    short = ro["hops"].astype(np.int64) + 1 <= 8
    hit = np.isin(wo, ch).any(axis=1)
    return int(np.where(short, hit, by_sum).sum())


def _workloads():
    return {"cfg1-dense": lambda: synth.cfg1(0, "dense"),
            "fat-tree-80-dense": lambda: synth.trace_workload(5, 8, 4, 24, 3000, 12, 200, variant="dense"),
            "fat-tree-320-rpath": lambda: synth.trace_workload(6, 16, 8, 300, 20000, 32, 4000)}


@pytest.mark.parametrize("name", list(_workloads()))
def test_first_call_matches_oracle(g, orc, name):
    wl = _workloads()[name]()
    rec, vs, wk, n, flags = _run(wl, wl["rule_off"], wl["rules"], None, None, None)
    ro, vo, wo, err = _oracle(orc, wl, wl["rule_off"], wl["rules"])
    _same_records(rec, ro)
    assert np.array_equal(vs, vo) and np.array_equal(wk, wo) and n == wl["ingress"].shape[0] and flags == err


@pytest.mark.parametrize("use_walk", [True, False])
@pytest.mark.parametrize("resize", [False, True])
@pytest.mark.parametrize("name", list(_workloads()))
def test_delta_from_oracle_state(g, orc, name, resize, use_walk):
    wl = _workloads()[name]()
    S = wl["S"]
    ro, vo, wo, _ = _oracle(orc, wl, wl["rule_off"], wl["rules"])
    changed = np.random.default_rng(3).choice(S, size=min(4, S), replace=False)
    r_off2, rules2 = synth.mutate_tables(3, wl["port_off"], wl["rule_off"], wl["rules"], changed, resize=resize)
    rec, vs, wk, n, flags = _run(wl, r_off2, rules2, ro, vo, changed, walk=wo, use_walk=use_walk)
    ro2, vo2, wo2, err2 = _oracle(orc, wl, r_off2, rules2)
    _same_records(rec, ro2)
    assert np.array_equal(vs, vo2) and flags == err2
    if use_walk:
        assert np.array_equal(wk, wo2)
    assert n == _expected_count(ro, vo, wo, changed, use_walk) and 0 < n < wl["ingress"].shape[0]


@pytest.mark.parametrize("name", ["fat-tree-80-dense", "fat-tree-320-rpath"])
def test_chained_deltas_on_gpu(g, orc, name):
    wl = _workloads()[name]()
    S = wl["S"]
    rule_off, rules = wl["rule_off"], wl["rules"]
    import paper_2602_16100_amd as pc
    ctx = pc.Context(0)  # one context: later calls re-prepare only the changed switches
    ctx.keep_tables(True)
    rec, vs, wk, _, _ = _run(wl, rule_off, rules, None, None, None, ctx=ctx)
    rng = np.random.default_rng(9)
    for step in range(4):
        changed = rng.choice(S, size=int(rng.integers(1, 6)), replace=True)  # repeats allowed
        rule_off, rules = synth.mutate_tables(20 + step, wl["port_off"], rule_off, rules, changed, resize=step % 2 == 1)
        rec, vs, wk, n, flags = _run(wl, rule_off, rules, rec, vs, changed, walk=wk, ctx=ctx)
        ro, vo, wo, err = _oracle(orc, wl, rule_off, rules)
        _same_records(rec, ro)
        assert np.array_equal(vs, vo) and np.array_equal(wk, wo) and flags == err


def test_chain_across_group_boundaries(g, orc):
    """Tables of exactly 32 rules per switch: resizing a switch to 31 or 33
    rules changes its number of 32-rule groups, so the kept tables cannot
    serve and every switch is prepared again; the next delta (sizes kept)
    re-prepares only its changed switch.  Every step equals the oracle."""
    import paper_2602_16100_amd as pc
    wl = synth.trace_workload(7, 8, 4, 32, 4000, 12, 300, variant="dense")
    ctx = pc.Context(0)
    ctx.keep_tables(True)
    rule_off, rules = wl["rule_off"], wl["rules"]
    rec, vs, wk, _, _ = _run(wl, rule_off, rules, None, None, None, ctx=ctx)
    for step, (sw, resize) in enumerate([([4, 9], True), ([30], False), ([4, 11, 70], True), ([5], False)]):
        rule_off, rules = synth.mutate_tables(40 + step, wl["port_off"], rule_off, rules, sw, resize=resize)
        rec, vs, wk, n, flags = _run(wl, rule_off, rules, rec, vs, np.array(sw, np.int32), walk=wk, ctx=ctx)
        ro, vo, wo, err = _oracle(orc, wl, rule_off, rules)
        _same_records(rec, ro)
        assert np.array_equal(vs, vo) and np.array_equal(wk, wo) and flags == err


def test_edge_cases(g, orc):
    wl = synth.trace_workload(5, 8, 4, 24, 3000, 12, 200, variant="dense")
    S, T = wl["S"], wl["ingress"].shape[0]
    ingress = wl["ingress"].copy()
    ingress[:4] = [-1, S, -7, 10 ** 6]  # invalid ingresses: MISS records, empty summaries and walks, SWITCH flag
    wl.arrays["ingress"] = ingress
    ro, vo, wo, err = _oracle(orc, wl, wl["rule_off"], wl["rules"])
    assert err == F_SWITCH and (vo[:4] == 0).all() and (wo[:4] == -1).all()
    rec, vs, wk, n, flags = _run(wl, wl["rule_off"], wl["rules"], None, None, None)
    _same_records(rec, ro)
    assert np.array_equal(vs, vo) and np.array_equal(wk, wo) and flags == F_SWITCH
    # no change: nothing traced again, nothing moves
    rec2, vs2, wk2, n, flags = _run(wl, wl["rule_off"], wl["rules"], ro, vo, np.zeros(0, np.int32), walk=wo)
    _same_records(rec2, ro)
    assert np.array_equal(vs2, vo) and np.array_equal(wk2, wo) and n == 0 and flags == F_SWITCH
    # out-of-range ids are ignored and flagged; a valid one still counts
    r_off2, rules2 = synth.mutate_tables(4, wl["port_off"], wl["rule_off"], wl["rules"], [17])
    ids = np.array([-1, 17, S, 17], np.int32)
    rec3, vs3, wk3, n, flags = _run(wl, r_off2, rules2, ro, vo, ids, walk=wo)
    ro3, vo3, wo3, err3 = _oracle(orc, wl, r_off2, rules2)
    _same_records(rec3, ro3)
    assert np.array_equal(vs3, vo3) and np.array_equal(wk3, wo3) and flags == err3 | F_SWITCH
    assert n == _expected_count(ro, vo, wo, [17])
    # every switch changed: every trace with a valid ingress is traced again
    r_off4, rules4 = synth.mutate_tables(5, wl["port_off"], wl["rule_off"], wl["rules"], np.arange(S), resize=True)
    rec4, vs4, wk4, n, flags = _run(wl, r_off4, rules4, ro, vo, np.arange(S, dtype=np.int32), walk=wo)
    ro4, vo4, wo4, _ = _oracle(orc, wl, r_off4, rules4)
    _same_records(rec4, ro4)
    assert np.array_equal(vs4, vo4) and np.array_equal(wk4, wo4) and n == T - 4
    # no traces
    wl0 = synth.trace_workload(5, 8, 4, 24, 3000, 12, 200, variant="dense")
    wl0.arrays["hdr"] = wl0["hdr"][:0]
    wl0.arrays["ingress"] = wl0["ingress"][:0]
    rec5, vs5, wk5, n, flags = _run(wl0, wl0["rule_off"], wl0["rules"], np.zeros(0, ro.dtype), np.zeros(0, np.uint64),
                                    np.array([3], np.int32), walk=np.zeros((0, 8), np.int32))
    assert n == 0 and rec5.shape[0] == 0


def test_delta_combined_workload_size(g, orc):
    """The combined workload's 699,050 traces over 2,880 switches of 16,384
    rules: a full first call, then the tables of one core, two aggregation
    and three edge switches rewritten.  Every record, summary and walk
    record equals a full GPU trace on the new tables; the traces traced
    again are exactly those whose walk visited a changed switch, except walks
    longer than their record (selected by summary bits); 4,000 sampled traces
    (half of them re-traced) equal the oracle."""
    import paper_2602_16100_amd as pc
    wl = synth.cfg5()
    ctx = pc.Context(0)
    ctx.keep_tables(True)
    rec, vs, wk, n, _ = _run(wl, wl["rule_off"], wl["rules"], None, None, None, ctx=ctx)
    k, h = 48, 24  # pod p: edge switches p*k + [0, h), aggregation p*k + [h, k); core from k*k
    changed = np.array([k * k + 5, 3 * k + h + 6, 10 * k + h + 16, 0, 5 * k + 2, 20 * k + 7], np.int32)
    assert changed.max() < wl["S"]
    r_off2, rules2 = synth.mutate_tables(8, wl["port_off"], wl["rule_off"], wl["rules"], changed)
    rec2, vs2, wk2, n2, flags = _run(wl, r_off2, rules2, rec, vs, changed, walk=wk, ctx=ctx)
    full, vfull, wfull, _, _ = _run(wl, r_off2, rules2, None, None, None)
    _same_records(rec2, full)
    assert np.array_equal(vs2, vfull) and np.array_equal(wk2, wfull) and flags == 0
    short = rec["hops"].astype(np.int64) + 1 <= 8
    assert short.mean() > 0.95  # nearly every walk fits its record
    assert n2 == _expected_count(rec, vs, wk, changed) and 0 < n2 < wl["ingress"].shape[0] // 10
    hit = np.flatnonzero(np.isin(wk, changed).any(axis=1) & short)
    rng = np.random.default_rng(4)
    idx = np.sort(np.concatenate([rng.choice(hit, min(2000, hit.shape[0]), replace=False),
                                  rng.choice(wl["ingress"].shape[0], 2000, replace=False)]))
    ro, vo, wo, err = _oracle(orc, wl, r_off2, rules2, idx=idx)
    _same_records(rec2[idx], ro)
    assert np.array_equal(vs2[idx], vo) and np.array_equal(wk2[idx], wo) and err == 0


@pytest.mark.parametrize("keep", [False, True])
def test_two_workloads_of_equal_size_on_one_context(g, orc, keep):
    """A delta chain on one workload, then a first call and a delta on a
    second workload with the same switch count, all on one context.  Without
    the keep-tables promise every call prepares anew; with it, the second
    workload's first call (C < 0) replaces the kept tables.  Either way the
    second workload's delta equals the oracle's full trace."""
    import paper_2602_16100_amd as pc
    wa = synth.trace_workload(11, 8, 4, 40, 3000, 12, 250, variant="dense")
    wb = synth.trace_workload(12, 8, 4, 40, 3000, 12, 250, variant="dense")
    assert wa["S"] == wb["S"]
    ctx = pc.Context(0)
    ctx.keep_tables(keep)
    rec, vs, wk, _, _ = _run(wa, wa["rule_off"], wa["rules"], None, None, None, ctx=ctx)
    ra, rules_a = synth.mutate_tables(3, wa["port_off"], wa["rule_off"], wa["rules"], [5, 9])
    _run(wa, ra, rules_a, rec, vs, np.array([5, 9], np.int32), walk=wk, ctx=ctx)
    # workload B: its results from the oracle, then a delta on the same context
    ro, vo, wo, _ = _oracle(orc, wb, wb["rule_off"], wb["rules"])
    if keep:  # the promise covers calls on the same tables: B starts with a full call
        rec_b, vs_b, wk_b, _, _ = _run(wb, wb["rule_off"], wb["rules"], None, None, None, ctx=ctx)
        _same_records(rec_b, ro)
    rb, rules_b = synth.mutate_tables(4, wb["port_off"], wb["rule_off"], wb["rules"], [7])
    rec2, vs2, wk2, n, flags = _run(wb, rb, rules_b, ro, vo, np.array([7], np.int32), walk=wo, ctx=ctx)
    ro2, vo2, wo2, err = _oracle(orc, wb, rb, rules_b)
    _same_records(rec2, ro2)
    assert np.array_equal(vs2, vo2) and np.array_equal(wk2, wo2) and flags == err


def test_default_context_prepares_every_call(g, orc):
    """Without the promise, a delta call on tables that differ from the
    context's previous call in unlisted switches as well still equals the
    oracle: every call prepares every switch.  (The previous results passed
    in are those of the tables' last version, as the delta contract asks.)"""
    import paper_2602_16100_amd as pc
    wl = synth.trace_workload(13, 8, 4, 40, 3000, 12, 250, variant="dense")
    ctx = pc.Context(0)
    _run(wl, wl["rule_off"], wl["rules"], None, None, None, ctx=ctx)          # the context's last tables: A
    r2, rules2 = synth.mutate_tables(6, wl["port_off"], wl["rule_off"], wl["rules"], [3, 17, 40])   # B
    rb, vb, wb_, _ = _oracle(orc, wl, r2, rules2)
    r3, rules3 = synth.mutate_tables(7, wl["port_off"], r2, rules2, [20, 21])                     # C
    rec3, vs3, wk3, n, flags = _run(wl, r3, rules3, rb, vb, np.array([20, 21], np.int32), walk=wb_, ctx=ctx)
    ro3, vo3, wo3, err3 = _oracle(orc, wl, r3, rules3)
    _same_records(rec3, ro3)
    assert np.array_equal(vs3, vo3) and np.array_equal(wk3, wo3) and flags == err3
    # the selected walks meet the switches that changed between A and B as well
    both = np.isin(wb_, [20, 21]).any(axis=1) & np.isin(wb_, [3, 17, 40]).any(axis=1)
    assert both.sum() > 0
