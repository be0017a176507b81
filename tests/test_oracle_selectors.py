"""Pins for the oracle's selector evaluation (placement constraints).

The paper fixes the semantics only through its examples: a placement
constraint is a node selector / affinity over node labels (Formal Model,
example intent), the 5-worker label matrix, and the fail-closed outcome of
a hallucinated label.  The operator semantics are Kubernetes node
affinity's.  Pins: the paper's label table, exhaustive set algebra on a
small schema, closed-form histograms at scale, lattice identities.
"""
import itertools

import numpy as np
import pytest

import synth
from helpers import bits_to_set, encode_label_matrix, encode_selector, load_golden


def test_paper_label_matrix(orc):
    fx = load_golden("paper_label_matrix.json")
    labels, vocab = encode_label_matrix(fx)
    names = [n["name"] for n in fx["nodes"]]
    for case in fx["cases"]:
        preds = encode_selector(fx, vocab, case["selector"])
        off = np.array([0, len(preds)], np.int32)
        feas, pc, err = orc.selectors(labels, off, preds)
        got = {names[n] for n in bits_to_set(feas[0], len(names))}
        assert got == set(case["expect"]), case["cite"]
        assert pc[0] == len(case["expect"])
        assert err == 0


def _all_nodes_schema():
    """2 labels, each value in {0, 1, 2, absent}: every assignment once (16 nodes)."""
    vals = [0, 1, 2, synth.ABSENT]
    return np.array(list(itertools.product(vals, vals)), np.uint8)


def _k8s_set(labels, label, op, S):
    """Node set of one predicate by Kubernetes node-affinity set semantics."""
    N = labels.shape[0]
    has = {n for n in range(N) if labels[n, label] != synth.ABSENT}
    member = {n for n in has if int(labels[n, label]) in S}
    if op == synth.OP_IN:
        return member
    if op == synth.OP_NOTIN:
        return set(range(N)) - member
    return has


def test_exhaustive_small_schema(orc):
    labels = _all_nodes_schema()
    N = labels.shape[0]
    subsets = [set(c) for r in range(4) for c in itertools.combinations(range(3), r)]
    single = []
    for l in range(2):
        for op in (synth.OP_IN, synth.OP_NOTIN):
            for S in subsets:
                single.append((l, op, S))
        single.append((l, synth.OP_EXISTS, set()))
    rows = [()] + [(p,) for p in single] + list(itertools.product(single, single))
    off = np.zeros(len(rows) + 1, np.int32)
    off[1:] = np.cumsum([len(r) for r in rows])
    preds = np.zeros(int(off[-1]), synth.PRED_DT)
    j = 0
    for r in rows:
        for (l, op, S) in r:
            preds[j]["label"] = l
            preds[j]["op"] = op
            preds[j]["vals"] = synth.values_to_bitmap(np.array([sorted(S) + [-1] * (4 - len(S))], np.int32))[0]
            j += 1
    feas, pc, err = orc.selectors(labels, off, preds)
    assert err == 0
    for i, r in enumerate(rows):
        want = set(range(N))
        for (l, op, S) in r:
            want &= _k8s_set(labels, l, op, S)
        assert bits_to_set(feas[i], N) == want, r
        assert pc[i] == len(want)


def test_closed_form_histograms(orc):
    """Single-predicate rows over a random cluster with absent labels:
    |In S| = sum of the label histogram over S, |NotIn S| = N - |In S|,
    |Exists| = N - #absent.  Ragged N (not a multiple of 64)."""
    rng = np.random.default_rng(11)
    N, L = 5000 + 37, 12
    cards = rng.choice([2, 4, 16, 64, 200], size=L)
    labels = synth.gen_labels(rng, N, cards, absent_p=0.07)
    off, preds = synth.gen_preds(rng, 600, cards, 1, 1)
    feas, pc, err = orc.selectors(labels, off, preds)
    assert err == 0
    W = (N + 63) // 64
    for i in range(600):
        p = preds[i]
        col = labels[:, p["label"]]
        hist = np.bincount(col, minlength=256)
        S = [v for v in range(255) if (int(p["vals"][v >> 6]) >> (v & 63)) & 1]
        n_in = int(hist[S].sum())
        want = {synth.OP_IN: n_in, synth.OP_NOTIN: N - n_in, synth.OP_EXISTS: N - int(hist[255])}[int(p["op"])]
        assert pc[i] == want
        # padding bits of the last word are zero
        tail = N - 64 * (W - 1)
        assert int(feas[i, W - 1]) >> tail == 0


def test_lattice_identities(orc):
    rng = np.random.default_rng(5)
    N, L = 3000, 6
    cards = np.array([2, 4, 16, 64, 8, 3])
    labels = synth.gen_labels(rng, N, cards, absent_p=0.05)
    rows = []
    for _ in range(80):
        l = int(rng.integers(0, L))
        S1 = set(int(x) for x in rng.choice(cards[l], size=min(3, cards[l]), replace=False))
        S2 = set(int(x) for x in rng.choice(cards[l], size=min(2, cards[l]), replace=False))
        rows.append((l, S1, S2))
    recs = []
    offs = [0]
    for (l, S1, S2) in rows:
        for spec in ([(l, 0, S1)], [(l, 1, S1)], [(l, 0, S1), (l, 0, S2)], [(l, 0, S1 & S2)]):
            for (ll, op, S) in spec:
                r = np.zeros(1, synth.PRED_DT)[0]
                r["label"], r["op"] = ll, op
                r["vals"] = synth.values_to_bitmap(np.array([sorted(S) + [-1] * (4 - len(S))], np.int32))[0]
                recs.append(r)
            offs.append(len(recs))
    preds = np.array(recs, synth.PRED_DT)
    off = np.array(offs, np.int32)
    feas, pc, err = orc.selectors(labels, off, preds)
    W = feas.shape[1]
    full = np.zeros(W, np.uint64)
    for n in range(N):
        full[n >> 6] |= np.uint64(1) << np.uint64(n & 63)
    for k in range(len(rows)):
        f_in, f_not, f_and, f_meet = feas[4 * k: 4 * k + 4]
        assert np.array_equal(f_in | f_not, full)           # In S or NotIn S = everything
        assert not np.any(f_in & f_not)                      # and never both
        assert np.array_equal(f_and, f_meet)                 # In S1 and In S2 = In (S1 & S2)
        assert np.array_equal(f_and & ~f_in, np.zeros(W, np.uint64))  # a conjunct never adds nodes


def test_empty_row_and_empty_sets(orc):
    labels = _all_nodes_schema()
    N = labels.shape[0]
    preds = np.zeros(2, synth.PRED_DT)
    preds[0]["op"] = synth.OP_IN
    preds[1]["op"] = synth.OP_NOTIN
    off = np.array([0, 0, 1, 2], np.int32)      # empty row, In {}, NotIn {}
    feas, pc, err = orc.selectors(labels, off, preds)
    assert list(pc) == [N, 0, N]


@pytest.mark.parametrize("field,value", [("label", 9), ("op", 3), ("rsv0", 1), ("rsv1", 7)])
def test_malformed_predicate(orc, field, value):
    labels = _all_nodes_schema()
    preds = np.zeros(1, synth.PRED_DT)
    preds[0]["op"] = synth.OP_EXISTS
    preds[0][field] = value
    off = np.array([0, 1], np.int32)
    feas, pc, err = orc.selectors(labels, off, preds)
    assert pc[0] == 0 and err & orc.F_PRED


def test_value_255_in_set_is_malformed(orc):
    labels = _all_nodes_schema()
    preds = np.zeros(1, synth.PRED_DT)
    preds[0]["op"] = synth.OP_NOTIN
    preds[0]["vals"][3] = np.uint64(1) << np.uint64(63)
    feas, pc, err = orc.selectors(labels, np.array([0, 1], np.int32), preds)
    assert pc[0] == 0 and err & orc.F_PRED


def test_bad_offsets(orc):
    labels = _all_nodes_schema()
    preds = np.zeros(2, synth.PRED_DT)
    preds["op"] = synth.OP_EXISTS
    off = np.array([0, 2, 1, 5], np.int32)      # row 1 decreasing, row 2 past the end
    feas, pc, err = orc.selectors(labels, off, preds)
    assert err & orc.F_OFFSETS
    assert pc[1] == 0 and pc[2] == 0


def test_row_subset_matches_full(orc):
    w = synth.selector_workload(3, 700, 10, 50, absent_p=0.02)
    f_all, p_all, _ = orc.selectors(w["labels"], w["pred_off"], w["preds"])
    rows = np.array([49, 0, 17, 17, 3], np.int32)
    f_sub, p_sub, _ = orc.selectors(w["labels"], w["pred_off"], w["preds"], rows=rows)
    assert np.array_equal(f_sub, f_all[rows]) and np.array_equal(p_sub, p_all[rows])


def test_hybrid_rows_hold_for_their_endpoints(orc):
    """The combined generator builds hybrid rows to admit both endpoints;
    only the misplaced destinations (1 in 16) may fall outside them."""
    w = synth.combined_workload(9, 1500, 16, 4, 2, 64, 3000)
    feas, pc, _ = orc.selectors(w["labels"], w["pred_off"], w["preds"])
    it = w["intents"]
    hyb = np.flatnonzero(it["kind"] == synth.KIND_HYBRID)
    dst_out = 0
    for i in hyb:
        r, a, b = int(it["sel_row"][i]), int(it["src_node"][i]), int(it["dst_node"][i])
        assert (int(feas[r, a >> 6]) >> (a & 63)) & 1
        dst_out += not ((int(feas[r, b >> 6]) >> (b & 63)) & 1)
    assert 0 < dst_out < hyb.shape[0] / 8
