"""Parity of pc_update_nodes (through the C ABI): after relabelling a set of
nodes, the in-place update of the GPU's own full evaluation equals the
GPU's full evaluation of the new labels and the oracle's update, bit-exact
(bitsets, popcounts, data-error word); node lists of 1 to 4,096 entries,
repeated, unsorted and out-of-range nodes, several 64-node batches sharing
bitset words, absent labels, malformed rows, and the combined workload's
full size."""
import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def g():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


@pytest.fixture(params=["default", "kernel"])
def path(request, monkeypatch):
    """default: the library's own switch to full re-evaluation above W/16
    nodes; kernel: the incremental kernels for every list size."""
    if request.param == "kernel":
        monkeypatch.setenv("PC_UPDATE_FULL_ABOVE", str(1 << 30))
    else:
        monkeypatch.delenv("PC_UPDATE_FULL_ABOVE", raising=False)
    return request.param


def _relabel(rng, labels, cards, nodes, absent_p=0.1):
    new = labels.copy()
    for n in np.unique(nodes):
        if 0 <= n < labels.shape[0]:
            row = rng.integers(0, np.asarray(cards)[None, :], size=(1, labels.shape[1]))[0].astype(np.uint8)
            row[rng.random(labels.shape[1]) < absent_p] = synth.ABSENT
            new[n] = row
    return new


def _gpu_update(labels_new, off, preds, nodes, f0, p0):
    import torch
    import paper_2602_16100_amd as pc
    ctx = pc.context()
    ctx.data_errors(clear=True)
    d = lambda a: pc.to_device(a, "cuda")  # noqa: E731
    f = torch.from_numpy(np.ascontiguousarray(f0).view(np.int64)).cuda()
    p = torch.from_numpy(np.ascontiguousarray(p0).view(np.int32)).cuda()
    pc.pc_update_nodes(d(labels_new), d(off), d(preds), d(np.ascontiguousarray(nodes, np.int32)), f, p)
    torch.cuda.synchronize()
    return f.cpu().numpy().view(np.uint64), p.cpu().numpy().view(np.uint32), ctx.data_errors(clear=True)


def _gpu_full(labels, off, preds):
    import gpu_run
    return gpu_run.selectors(labels, off, preds)


@pytest.mark.parametrize("M,clustered", [(1, False), (5, True), (64, False), (65, True), (700, False),
                                         (4096, True)])
def test_update_matches_full_evaluation(g, orc, path, M, clustered):
    wl = synth.selector_workload(7, 9000 + 13, 16, 1500, card_choices=(2, 3, 16, 64, 200), absent_p=0.05)
    labels, off, preds = wl["labels"], wl["pred_off"], wl["preds"]
    rng = np.random.default_rng(M)
    f0, p0 = _gpu_full(labels, off, preds)
    if clustered:  # many nodes per bitset word, words straddling 64-node batches
        nodes = (rng.integers(0, 9000 // 40, size=M) * 40 + rng.integers(0, 40, size=M)).astype(np.int32)
    else:
        nodes = rng.integers(0, 9013, size=M).astype(np.int32)
    if M > 2:
        nodes[2] = nodes[0]
    new = _relabel(rng, labels, wl.meta["cards"], nodes)
    fu, pu, eu = _gpu_update(new, off, preds, nodes, f0, p0)
    ff, pf = _gpu_full(new, off, preds)
    fo, po, eo = orc.update_nodes(new, off, preds, nodes, f0, p0)
    assert eu == eo == 0
    assert np.array_equal(fu, ff) and np.array_equal(pu, pf)
    assert np.array_equal(fu, fo) and np.array_equal(pu, po)


def test_update_out_of_range_and_malformed(g, orc, path):
    wl = synth.selector_workload(8, 3000, 6, 300, absent_p=0.1)
    labels, off, preds = wl["labels"], wl["pred_off"].copy(), wl["preds"].copy()
    preds[5]["op"] = 7
    off[11] = off[12] + 2
    f0, p0 = _gpu_full(labels, off, preds)
    rng = np.random.default_rng(3)
    nodes = np.array([17, -4, 3000, 2999, 17, 0, 1 << 30], np.int32)
    new = _relabel(rng, labels, wl.meta["cards"], nodes)
    fu, pu, eu = _gpu_update(new, off, preds, nodes, f0, p0)
    fo, po, eo = orc.update_nodes(new, off, preds, nodes, f0, p0)
    assert eu == eo == 1 | 2 | 128
    assert np.array_equal(fu, fo) and np.array_equal(pu, po)
    # an empty list changes nothing (flags of the rows still raised)
    fu, pu, eu = _gpu_update(labels, off, preds, np.zeros(0, np.int32), f0, p0)
    assert eu == 3 and np.array_equal(fu, f0) and np.array_equal(pu, p0)


def test_update_full_size(g, orc, path):
    """The combined workload's cluster and selector rows (699,051 rows x
    50,000 nodes): 64 relabelled nodes; the update equals the full
    evaluation of the new labels."""
    wl = synth.cfg5()
    labels, off, preds = wl["labels"], wl["pred_off"], wl["preds"]
    f0, p0 = _gpu_full(labels, off, preds)
    rng = np.random.default_rng(64)
    nodes = rng.integers(0, 50000, size=64).astype(np.int32)
    new = _relabel(rng, labels, wl.meta["cards"], nodes, absent_p=0.0)
    fu, pu, eu = _gpu_update(new, off, preds, nodes, f0, p0)
    ff, pf = _gpu_full(new, off, preds)
    assert eu == 0
    assert np.array_equal(pu, pf)
    assert np.array_equal(fu, ff)
    assert not np.array_equal(pu, p0)
