"""The seeded generators produce the stated shapes and statistics."""
import numpy as np
import pytest

import synth


@pytest.mark.parametrize("k,S,links", [(4, 20, 32), (32, 1280, 16384), (48, 2880, 55296)])
def test_fat_tree_counts_and_symmetry(k, S, links):
    t = synth.fat_tree(k, 8)
    assert t["S"] == S and t["H"] == k ** 3 // 4
    peer, off = t["port_peer"], t["port_off"]
    assert int((peer >= 0).sum()) == 2 * links
    # every link is seen from both ends
    src = np.repeat(np.arange(S), np.diff(off))
    m = peer >= 0
    fwd = set(zip(src[m].tolist(), peer[m].tolist()))
    assert all((v, u) in fwd for (u, v) in fwd)
    assert t["adj"].shape[0] == 2 * links


def test_care_bit_fraction():
    rng = np.random.default_rng(0)
    w = synth.care_bits(rng, (200_000,), 0.7)
    frac = np.unpackbits(w.view(np.uint8)).mean()
    assert abs(frac - 717 / 1024) < 0.002


def test_distinct_values():
    rng = np.random.default_rng(1)
    card = rng.choice([2, 4, 16, 64], size=20000)
    m = np.minimum(rng.integers(1, 5, size=20000), card)
    v = synth.distinct_values(rng, card, m)
    for i in range(2000):
        got = v[i][v[i] >= 0]
        assert len(got) == m[i] and len(set(got.tolist())) == m[i] and np.all(got < card[i])


def test_rgg_degree():
    wl = synth.rgg_workload(0, 200_000, 16, 4)
    mean_deg = wl["adj"].shape[0] / wl["V"]
    assert abs(mean_deg - 4.0) < 0.05
    assert wl["region"].max() < 16


def test_combined_class_split():
    I = 1_048_576
    kinds = np.array([1, 2, 3])[np.arange(I) % 3]
    assert list(np.bincount(kinds)[1:]) == [349_526, 349_525, 349_525]
    wl = synth.combined_workload(1, 500, 8, 4, 2, 64, 100)
    assert list(np.bincount(wl["intents"]["kind"])[1:]) == [34, 33, 33]


def test_rpath_table_fill():
    wl = synth.trace_workload(2, 8, 4, 256, 1000, 32, 2000)
    assert wl.meta["path_rules_dropped"] == 0
    r = wl["rules"]
    # distinct priorities per switch
    for s in range(wl["S"]):
        p = r["priority"][wl["rule_off"][s]:wl["rule_off"][s + 1]]
        assert np.unique(p).shape[0] == p.shape[0]
    # canonical values: no bit outside the mask
    assert not np.any(r["value"] & ~r["mask"])
    assert not np.any(r["mask"][:, 3] >> 8)
    drop = np.mean(r["action"] == synth.DROP)
    assert 0.04 < drop < 0.06
