"""Pins of the CPU oracle's incremental re-evaluation after node-label
changes: the updated bitsets and popcounts equal a full evaluation of the
new labels by the separately pinned selector oracle, for random changes,
repeated and unsorted node lists, absent labels and malformed rows; an
empty list changes nothing; nodes outside [0, N) are skipped and flagged."""
import numpy as np
import pytest

import synth


def _relabel(rng, labels, cards, nodes, absent_p=0.1):
    new = labels.copy()
    for n in np.unique(nodes):
        if n < 0 or n >= labels.shape[0]:
            continue
        row = rng.integers(0, np.asarray(cards)[None, :], size=(1, labels.shape[1]))[0].astype(np.uint8)
        row[rng.random(labels.shape[1]) < absent_p] = synth.ABSENT
        new[n] = row
    return new


@pytest.mark.parametrize("M", [1, 7, 64, 65, 300])
def test_update_equals_full_evaluation(orc, M):
    wl = synth.selector_workload(3, 3000 + 11, 10, 500, card_choices=(2, 3, 16, 64), absent_p=0.05)
    labels, off, preds = wl["labels"], wl["pred_off"], wl["preds"]
    rng = np.random.default_rng(M)
    f0, p0, e0 = orc.selectors(labels, off, preds)
    nodes = rng.integers(0, labels.shape[0], size=M).astype(np.int32)
    if M > 1:
        nodes[1] = nodes[0]  # a repeated node
    new = _relabel(rng, labels, wl.meta["cards"], nodes)
    f1, p1, e1 = orc.update_nodes(new, off, preds, nodes, f0, p0)
    ff, pf, ef = orc.selectors(new, off, preds)
    assert e1 == e0 == ef == 0
    assert np.array_equal(f1, ff) and np.array_equal(p1, pf)
    assert not np.array_equal(f1, f0) or M == 1


def test_update_no_nodes_and_out_of_range(orc):
    wl = synth.selector_workload(4, 700, 6, 80, absent_p=0.1)
    labels, off, preds = wl["labels"], wl["pred_off"], wl["preds"]
    f0, p0, _ = orc.selectors(labels, off, preds)
    f1, p1, e1 = orc.update_nodes(labels, off, preds, np.zeros(0, np.int32), f0, p0)
    assert e1 == 0 and np.array_equal(f1, f0) and np.array_equal(p1, p0)
    rng = np.random.default_rng(0)
    nodes = np.array([5, -1, 700, 9], np.int32)
    new = _relabel(rng, labels, wl.meta["cards"], nodes)
    f1, p1, e1 = orc.update_nodes(new, off, preds, nodes, f0, p0)
    ff, pf, _ = orc.selectors(new, off, preds)
    assert e1 == 128 and np.array_equal(f1, ff) and np.array_equal(p1, pf)


def test_update_malformed_rows(orc):
    """Malformed rows and predicates keep the full evaluation's meaning
    (empty rows) and flags."""
    wl = synth.selector_workload(8, 500, 6, 40)
    labels, off, preds = wl["labels"], wl["pred_off"].copy(), wl["preds"].copy()
    preds[3]["op"] = 9
    off[7] = off[8] + 1  # bad pairs for rows 6 and 7
    f0, p0, e0 = orc.selectors(labels, off, preds)
    rng = np.random.default_rng(1)
    nodes = rng.integers(0, 500, size=20).astype(np.int32)
    new = _relabel(rng, labels, wl.meta["cards"], nodes)
    f1, p1, e1 = orc.update_nodes(new, off, preds, nodes, f0, p0)
    ff, pf, ef = orc.selectors(new, off, preds)
    assert e1 == ef == e0 == 3
    assert np.array_equal(f1, ff) and np.array_equal(p1, pf)


def test_probes_are_bits_of_the_bitset(orc):
    """Membership probes equal the bits of the (separately pinned) full
    bitset; out-of-range rows or nodes answer 0 and raise NODE."""
    wl = synth.selector_workload(11, 2000 + 9, 8, 400, card_choices=(2, 5, 30), absent_p=0.1)
    labels, off, preds = wl["labels"], wl["pred_off"], wl["preds"]
    f, _, _ = orc.selectors(labels, off, preds)
    rng = np.random.default_rng(5)
    rows = rng.integers(0, 400, size=3000).astype(np.int32)
    nodes = rng.integers(0, 2009, size=3000).astype(np.int32)
    bits, err = orc.probes(labels, off, preds, rows, nodes)
    want = (f[rows, nodes >> 6] >> (nodes & 63).astype(np.uint64)) & np.uint64(1)
    assert err == 0 and np.array_equal(bits, want.astype(np.uint8))
    assert 0 < bits.sum() < 3000
    bits, err = orc.probes(labels, off, preds, np.array([0, -1, 400, 3], np.int32),
                           np.array([-2, 0, 0, 2009], np.int32))
    assert err == 128 and bits.tolist() == [0, 0, 0, 0]
