"""Parity of the verdict-only path (through the C ABI): popcounts without
the bitset (pc_eval_selectors_count), membership probes
(pc_probe_selectors) and the verdict from both (pc_report_counts) equal the
full path and the oracle, bit-exact, including the data-error word; at
small sizes with absent labels, malformed rows and intents, and on the
combined workload at full size."""
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


def _d(a):
    import paper_2602_16100_amd as pc
    return pc.to_device(a, "cuda")


def _count(labels, off, preds):
    import torch
    import paper_2602_16100_amd as pc
    ctx = pc.context()
    ctx.data_errors(clear=True)
    p = pc.pc_eval_selectors_count(_d(labels), _d(off), _d(preds))
    torch.cuda.synchronize()
    return p.cpu().numpy().view(np.uint32), ctx.data_errors(clear=True)


def _probe(labels, off, preds, rows, nodes):
    import torch
    import paper_2602_16100_amd as pc
    ctx = pc.context()
    ctx.data_errors(clear=True)
    b = pc.pc_probe_selectors(_d(labels), _d(off), _d(preds), _d(np.asarray(rows, np.int32)),
                              _d(np.asarray(nodes, np.int32)))
    torch.cuda.synchronize()
    return b.cpu().numpy(), ctx.data_errors(clear=True)


@pytest.mark.parametrize("seed,N", [(0, 5037), (1, 200), (2, 64 * 300 + 1)])
def test_count_and_probes(g, orc, seed, N):
    wl = synth.selector_workload(seed, N, 12, 800, card_choices=(2, 3, 16, 64, 200), absent_p=0.05)
    labels, off, preds = wl["labels"], wl["pred_off"].copy(), wl["preds"].copy()
    preds[4]["op"] = 5  # malformed for plain selectors
    off[9] = off[10] + 1
    pc_, e_c = _count(labels, off, preds)
    fo, po, eo = orc.selectors(labels, off, preds)
    assert np.array_equal(pc_, po) and e_c == eo
    rng = np.random.default_rng(seed)
    rows = rng.integers(-3, 803, size=5000)
    nodes = rng.integers(-3, N + 3, size=5000)
    bg, eg = _probe(labels, off, preds, rows, nodes)
    bo, eo2 = orc.probes(labels, off, preds, rows, nodes)
    assert np.array_equal(bg, bo) and eg == eo2


def _verdict_only(g, wl):
    """count + probes + pc_report_counts on the GPU."""
    import torch
    import paper_2602_16100_amd as pc
    it = wl["intents"]
    I = it.shape[0]
    p, _ = _count(wl["labels"], wl["pred_off"], wl["preds"])
    hyb = it["kind"] == 3
    rows = np.where(np.repeat(hyb, 2), np.repeat(it["sel_row"], 2), -1).astype(np.int32)
    nodes = np.stack([it["src_node"], it["dst_node"]], axis=1).reshape(-1).astype(np.int32)
    ends = np.zeros(2 * I, np.uint8)
    if hyb.any():
        sel = np.repeat(hyb, 2)
        b, _ = _probe(wl["labels"], wl["pred_off"], wl["preds"], rows[sel], nodes[sel])
        ends[sel] = b
    tr = g.trace(wl["S"], wl["port_off"], wl["port_peer"], wl["jur"], wl["rule_off"], wl["rules"], wl["hdr"],
                 wl["ingress"], wl["ttl"])
    rc = g.reach(wl["V"], wl["adj_off"], wl["adj"], wl["region"], wl["src"], wl["allowed"], wl["target"])
    ps, rs, sm = pc.pc_report_counts(_d(it), torch.from_numpy(p.view(np.int32)).cuda(), wl["N"], _d(ends),
                                     torch.from_numpy(np.ascontiguousarray(tr).view(np.uint8).reshape(-1, 12)).cuda(),
                                     _d(wl["expect"]), torch.from_numpy(rc.astype(np.int32)).cuda())
    torch.cuda.synchronize()
    return ps.cpu().numpy().view(np.uint64), rs.cpu().numpy(), pc.records(sm, pc.SUMMARY_DT)[0]


@pytest.mark.parametrize("make", ["cfg1", "combined", "malformed"])
def test_verdict_only_equals_full(g, orc, make):
    if make == "cfg1":
        wl = synth.cfg1(0)
    else:
        wl = synth.combined_workload(3, 3000 + 37, 16, 8, 4, 700, 3001)
        if make == "malformed":
            it = wl["intents"].copy()
            it["kind"][5] = 9
            it["src_node"][8] = -1 if it["kind"][8] == 3 else it["src_node"][8]
            it["sel_row"][14] = 1 << 30
            wl.arrays["intents"] = it
    pv, rv, sv = _verdict_only(g, wl)
    oo = orc.run_workload(wl)
    assert np.array_equal(pv, oo["pass"])
    assert np.array_equal(rv, oo["reason"])
    assert np.array_equal(sv.tobytes(), oo["summary"].tobytes())


def test_verdict_only_full_size(g, orc):
    """The combined workload at full size: the verdict-only path equals the
    full path's verdict (pass bits, reasons, summary)."""
    import torch
    import paper_2602_16100_amd as pc
    wl = synth.cfg5()
    full = g.run_workload(wl)
    pv, rv, sv = _verdict_only(g, wl)
    assert np.array_equal(pv, full["pass"])
    assert np.array_equal(rv, full["reason"])
    assert np.array_equal(sv.tobytes(), full["summary"].tobytes())
    p, _ = _count(wl["labels"], wl["pred_off"], wl["preds"])
    assert np.array_equal(p, full["popcnt"])
