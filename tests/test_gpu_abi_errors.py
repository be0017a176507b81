"""Boundary errors on a live context: argument errors return PC_EINVAL
before any device work is queued (outputs keep their sentinel, the
per-kernel profiler records no launch), and a refused scratch allocation
returns PC_ENOMEM, after which the same context works normally."""
import ctypes
import os

import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu

SENT = 0x5A


@pytest.fixture(scope="module")
def pc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2602_16100_amd as pc
    return pc


@pytest.fixture()
def live(pc):
    """A fresh context with profiling on, plus sentinel-filled device buffers."""
    import torch
    ctx = pc.Context(0)
    L = pc.lib()
    assert L.pc_profile(ctx.handle, 1) == pc.PC_OK
    bufs = {k: torch.full((n,), SENT, dtype=torch.uint8, device="cuda")
            for k, n in (("a", 4096), ("b", 4096), ("c", 4096), ("d", 4096), ("e", 4096), ("f", 4096),
                         ("out", 65536), ("out2", 65536), ("out3", 4096))}
    torch.cuda.synchronize()
    yield ctx, L, bufs
    del ctx


def _no_device_work(pc, ctx, L, bufs):
    import torch
    torch.cuda.synchronize()
    for k, b in bufs.items():
        assert bool((b == SENT).all()), f"buffer {k} was written"
    name = ctx_name = ctypes.c_char_p()
    n = ctypes.c_int64()
    ms = ctypes.c_double()
    assert L.pc_profile_read(ctx.handle, 0, ctypes.byref(name), ctypes.byref(n), ctypes.byref(ms)) == pc.PC_EINVAL, \
        f"a kernel was launched: {ctx_name.value}"


def _p(t):
    return ctypes.c_void_p(t.data_ptr())


def _cases(b):
    """(entry point, argument tuple after ctx) pairs, each with exactly one argument error."""
    a, bb, c, d, e, f, o, o2, o3 = (_p(b[k]) for k in ("a", "b", "c", "d", "e", "f", "out", "out2", "out3"))
    N0 = None
    sel = lambda N=64, L=8, I=4, n_preds=4, labels=a, pred_off=bb, preds=c, feas=o, pop=o2: \
        ("pc_eval_selectors", (labels, N, L, pred_off, preds, n_preds, I, feas, pop, N0))
    tr = lambda S=4, pp=bb, n_ports=16, jur=c, ro=d, rules=e, n_rules=16, hdr=f, ing=o3, T=8, ttl=16, out=o: \
        ("pc_trace_flows", (S, a, pp, n_ports, jur, ro, rules, n_rules, hdr, ing, T, ttl, out, N0))
    trw = lambda K=3, watch=o2, visit=o3, ttl=16: \
        ("pc_trace_flows_watch", (4, a, bb, 16, c, d, e, 16, f, o3, 8, ttl, watch, K, o, visit, N0))
    rc = lambda V=16, n_adj=32, Q=4, dist=o, src=bb: \
        ("pc_masked_reach", (V, a, bb, n_adj, c, Q, src, d, N0, dist, N0))
    rv = lambda Kv=1, Kf=2, via=e, forbid=f: \
        ("pc_masked_reach_via", (16, a, bb, 32, c, 4, d, e, f, via, Kv, forbid, Kf, o, N0))
    rp = lambda I=4, rows=4, W=1, N=64, T=4, Q=4, pss=o, reason=o2, summ=o3: \
        ("pc_report", (I, a, rows, bb, W, c, N, d, T, e, f, Q, pss, reason, summ, N0))
    up = lambda M=4, nodes=o3: \
        ("pc_update_nodes", (a, 64, 8, bb, c, 4, 4, nodes, M, o, o2, N0))
    syn = lambda V=16, max_hops=32, prio=100, Kv=1, Kf=1: \
        ("pc_synthesize_paths", (V, a, bb, 32, N0, c, 4, d, e, f, o3, Kv, o3, Kf, o2, o3, prio, max_hops, o, o2,
                                 o3, N0))
    return [
        ("selectors N<0", sel(N=-1)), ("selectors I<0", sel(I=-1)), ("selectors n_preds<0", sel(n_preds=-1)),
        ("selectors L=65536", sel(L=65536)), ("selectors L<0", sel(L=-1)),
        ("selectors L=0 with predicates", sel(L=0)), ("selectors null feasible", sel(feas=N0)),
        ("selectors null popcnt", sel(pop=N0)), ("selectors null pred_off", sel(pred_off=N0)),
        ("selectors null labels", sel(labels=N0)), ("selectors null preds", sel(preds=N0)),
        ("trace S<0", tr(S=-1)), ("trace T<0", tr(T=-1)), ("trace n_ports<0", tr(n_ports=-1)),
        ("trace n_rules<0", tr(n_rules=-1)), ("trace ttl=256", tr(ttl=256)), ("trace ttl<0", tr(ttl=-1)),
        ("trace null out", tr(out=N0)), ("trace null hdr", tr(hdr=N0)), ("trace null ingress", tr(ing=N0)),
        ("trace null rules", tr(rules=N0)), ("trace null port_peer", tr(pp=N0)), ("trace null jur", tr(jur=N0)),
        ("trace null rule_off", tr(ro=N0)),
        ("watch K=33", trw(K=33)), ("watch K<0", trw(K=-1)), ("watch null list", trw(watch=N0)),
        ("watch null visit", trw(visit=N0)), ("watch ttl=256", trw(ttl=256)),
        ("reach V<0", rc(V=-1)), ("reach Q<0", rc(Q=-1)), ("reach n_adj<0", rc(n_adj=-1)),
        ("reach null dist", rc(dist=N0)), ("reach null src", rc(src=N0)),
        ("via Kv=33", rv(Kv=33)), ("via Kf=33", rv(Kf=33)), ("via Kv<0", rv(Kv=-1)), ("via null via", rv(via=N0)),
        ("via null forbid", rv(forbid=N0)),
        ("report I<0", rp(I=-1)), ("report W too small", rp(W=1, N=65)), ("report N<0", rp(N=-1)),
        ("report null summary", rp(summ=N0)), ("report null pass", rp(pss=N0)),
        ("report null reason", rp(reason=N0)), ("report T<0", rp(T=-1)), ("report Q<0", rp(Q=-1)),
        ("update M=4097", up(M=4097)), ("update M<0", up(M=-1)), ("update null nodes", up(nodes=N0)),
        ("synthesize V above the LDS limit", syn(V=12289)), ("synthesize max_hops=256", syn(max_hops=256)),
        ("synthesize prio=65536", syn(prio=65536)), ("synthesize Kv=33", syn(Kv=33)),
        ("synthesize Kf=33", syn(Kf=33)),
    ]


def test_einval_with_live_context(pc, live):
    ctx, L, bufs = live
    cases = _cases(bufs)
    for name, (fn, args) in cases:
        rc = getattr(L, fn)(ctx.handle, *args)
        assert rc == pc.PC_EINVAL, f"{name}: returned {rc}"
        msg = L.pc_last_error(ctx.handle)
        assert msg and fn.encode() in msg, f"{name}: message {msg!r}"
    _no_device_work(pc, ctx, L, bufs)
    # the context is still usable: one valid call afterwards runs and is right
    import gpu_run
    assert L.pc_profile(ctx.handle, 0) == pc.PC_OK
    wl = synth.selector_workload(3, 300, 6, 20)
    import torch
    f, p = pc.pc_eval_selectors(gpu_run.dev(wl["labels"]), gpu_run.dev(wl["pred_off"]), gpu_run.dev(wl["preds"]),
                                ctx=ctx)
    torch.cuda.synchronize()
    pop = np.unpackbits(f.cpu().numpy().view(np.uint8), axis=1).sum(1)
    assert np.array_equal(pop, p.cpu().numpy().view(np.uint32))


def test_data_errors_null_flags(pc, live):
    ctx, L, bufs = live
    assert L.pc_data_errors(ctx.handle, None, None, 0) == pc.PC_EINVAL


def test_enomem_on_refused_scratch(pc, orc):
    """PC_FAIL_ALLOC refuses every scratch growth: a fresh context's first
    call that needs scratch returns PC_ENOMEM with a message; once the hook
    is off the same context computes the oracle's result."""
    import torch
    import gpu_run
    wl = synth.selector_workload(4, 1000, 8, 50)
    labels, off, preds = (gpu_run.dev(wl["labels"]), gpu_run.dev(wl["pred_off"]), gpu_run.dev(wl["preds"]))
    tw = synth.cfg1(0)
    ctx = pc.Context(0)
    os.environ["PC_FAIL_ALLOC"] = "1"
    try:
        with pytest.raises(pc.PCError) as ei:
            pc.pc_eval_selectors(labels, off, preds, ctx=ctx)
        assert ei.value.code == pc.PC_ENOMEM and "PC_FAIL_ALLOC" in str(ei.value)
        with pytest.raises(pc.PCError) as ei:
            pc.pc_trace_flows(tw["S"], gpu_run.dev(tw["port_off"]), gpu_run.dev(tw["port_peer"]),
                              gpu_run.dev(tw["jur"]), gpu_run.dev(tw["rule_off"]), gpu_run.dev(tw["rules"]),
                              gpu_run.dev(tw["hdr"]), gpu_run.dev(tw["ingress"]), tw["ttl"], ctx=ctx)
        assert ei.value.code == pc.PC_ENOMEM
    finally:
        del os.environ["PC_FAIL_ALLOC"]
    torch.cuda.synchronize()
    f, p = pc.pc_eval_selectors(labels, off, preds, ctx=ctx)
    torch.cuda.synchronize()
    fo, po, _ = orc.selectors(wl["labels"], wl["pred_off"], wl["preds"])
    assert np.array_equal(f.cpu().numpy().view(np.uint64), fo)
    assert np.array_equal(p.cpu().numpy().view(np.uint32), po)
