"""Pins of the CPU oracle's required node affinity (rows = OR of terms,
terms = AND of expressions, six operators, label-inventory flags).

The affinity oracle is checked against things it does not compute itself:
- the paper's 5-worker label matrix with hand-derived answers (golden
  fixture);
- reductions to the separately pinned selector oracle: every expression
  rewritten as an equivalent In / NotIn / Exists predicate (Gt t = In of
  the values above t, Lt t = In of the values below t, DoesNotExist = NotIn
  of every value), every term evaluated as a selector row, and the terms
  OR-ed with numpy;
- set algebra (DoesNotExist and Exists partition the nodes);
- numpy's unique values per label column for the inventory flags;
- closed forms for empty rows, empty terms and malformed inputs.
"""
import json
import os

import numpy as np
import pytest

import synth

HERE = os.path.dirname(os.path.abspath(__file__))
OPS = {"In": 0, "NotIn": 1, "Exists": 2, "DoesNotExist": 3, "Gt": 4, "Lt": 5}


def _bits(feas, N):
    return np.unpackbits(feas.view(np.uint8), bitorder="little", axis=-1)[..., :N].astype(bool)


def _pred(label, op, vals=(), thr=None):
    p = np.zeros(1, synth.PRED_DT)[0]
    p["label"] = label
    p["op"] = op
    bm = [0, 0, 0, 0]
    for v in vals:
        bm[int(v) >> 6] |= 1 << (int(v) & 63)
    if thr is not None:
        bm = [int(np.int64(thr).view(np.uint64)), 0, 0, 0]
    p["vals"] = np.array(bm, np.uint64)
    return p


def _csr(rows):
    """rows: list of rows, a row a list of terms, a term a list of preds."""
    row_off = [0]
    term_off = [0]
    preds = []
    for row in rows:
        for term in row:
            preds.extend(term)
            term_off.append(len(preds))
        row_off.append(len(term_off) - 1)
    arr = np.array(preds, synth.PRED_DT) if preds else np.zeros(0, synth.PRED_DT)
    return np.array(row_off, np.int32), np.array(term_off, np.int32), arr


def test_paper_label_matrix_affinity(orc):
    fx = json.load(open(os.path.join(HERE, "golden", "paper_affinity.json")))
    keys = fx["keys"]
    nodes = fx["nodes"]
    names = [n["name"] for n in nodes]
    # per key: carried values sorted -> codes 0.., values no node carries get the next codes
    codes = {}
    for k in keys:
        carried = sorted({n[k] for n in nodes if k in n})
        codes[k] = {v: i for i, v in enumerate(carried)}
    for case in fx["cases"]:
        for term in case["terms"]:
            for k, _, vals in term:
                for v in vals:
                    codes[k].setdefault(v, len(codes[k]))
    labels = np.full((len(nodes), len(keys)), synth.ABSENT, np.uint8)
    for i, n in enumerate(nodes):
        for j, k in enumerate(keys):
            if k in n:
                labels[i, j] = codes[k][n[k]]
    rows = []
    for case in fx["cases"]:
        rows.append([[_pred(keys.index(k), OPS[op], [codes[k][v] for v in vals]) for k, op, vals in term]
                     for term in case["terms"]])
    row_off, term_off, preds = _csr(rows)
    feas, pc, unk, err = orc.affinity(labels, row_off, term_off, preds)
    assert err == 0
    got = _bits(feas, len(nodes))
    for r, case in enumerate(fx["cases"]):
        assert sorted(np.array(names)[got[r]].tolist()) == sorted(case["expect"]), case["cite"]
        assert int(unk[r]) == case["unknown"], case["cite"]
        assert int(pc[r]) == len(case["expect"])


def _as_selector_pred(p, card_max=255):
    """The In / NotIn / Exists predicate equivalent to an affinity
    expression under the Kubernetes definitions."""
    op = int(p["op"])
    q = p.copy()
    if op <= 2:
        return q
    if op == 3:  # DoesNotExist: the label is absent = NotIn of every value
        vals = range(0, 255)
        q = _pred(int(p["label"]), 1, vals)
    else:
        t = int(np.uint64(p["vals"][0]).view(np.int64))
        vals = [v for v in range(0, 255) if (v > t if op == 4 else v < t)]
        q = _pred(int(p["label"]), 0, vals)
    return q


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_terms_reduce_to_selector_rows(orc, seed):
    """Each row = OR over its terms of the term's conjunction; each term
    is evaluated as a selector row after rewriting its expressions."""
    wl = synth.affinity_workload(seed, 700 + 13 * seed, 6, 150, card_choices=(2, 5, 16, 40), absent_p=0.15,
                                 tmin=0, tmax=4, kmin=0, kmax=4)
    labels, row_off, term_off, preds = wl["labels"], wl["row_off"], wl["term_off"], wl["preds"]
    N = labels.shape[0]
    feas, pc, unk, err = orc.affinity(labels, row_off, term_off, preds)
    assert err == 0
    sel = np.array([_as_selector_pred(p) for p in preds], synth.PRED_DT) if preds.shape[0] else preds
    tf, tp, terr = orc.selectors(labels, term_off, sel)
    assert terr == 0
    tbits = _bits(tf, N)
    empty_term = np.diff(term_off) == 0
    tbits[empty_term] = False  # an empty term matches no node (an empty selector row matches all)
    got = _bits(feas, N)
    for i in range(row_off.shape[0] - 1):
        b, e = row_off[i], row_off[i + 1]
        want = np.ones(N, bool) if b == e else tbits[b:e].any(axis=0)
        assert np.array_equal(got[i], want), f"row {i}"
    assert np.array_equal(pc, got.sum(axis=1))
    # the workload exercises every operator, empty rows and empty terms
    assert set(np.unique(preds["op"])) == set(range(6))
    assert (np.diff(row_off) == 0).any() and empty_term.any()


def test_gt_lt_thresholds_exhaustive(orc):
    """Gt / Lt at every threshold from -3 to 258 against the In set of the
    values above / below it, including absent labels (never admitted)."""
    rng = np.random.default_rng(5)
    N = 600
    labels = np.stack([rng.integers(0, 255, N), rng.integers(0, 7, N)], axis=1).astype(np.uint8)
    labels[rng.random(labels.shape) < 0.1] = synth.ABSENT
    rows = []
    for lab in range(2):
        for t in range(-3, 259):
            for op in (4, 5):
                rows.append([[_pred(lab, op, thr=t)]])
    row_off, term_off, preds = _csr(rows)
    feas, pc, _, err = orc.affinity(labels, row_off, term_off, preds)
    assert err == 0
    got = _bits(feas, N)
    x = labels.astype(np.int64)
    r = 0
    for lab in range(2):
        for t in range(-3, 259):
            for op in (4, 5):
                present = x[:, lab] != synth.ABSENT
                want = present & ((x[:, lab] > t) if op == 4 else (x[:, lab] < t))
                assert np.array_equal(got[r], want), (lab, t, op)
                r += 1


def test_doesnotexist_partitions_with_exists(orc):
    wl = synth.affinity_workload(3, 1000 + 7, 9, 1, absent_p=0.3)
    labels = wl["labels"]
    N, L = labels.shape
    labels[:, 4] = synth.ABSENT  # a label no node carries
    labels[:, 5] = 1  # a label every node carries
    rows = [[[_pred(l, 2)]] for l in range(L)] + [[[_pred(l, 3)]] for l in range(L)]
    row_off, term_off, preds = _csr(rows)
    feas, pc, unk, err = orc.affinity(labels, row_off, term_off, preds)
    assert err == 0
    b = _bits(feas, N)
    ex, dne = b[:L], b[L:]
    assert not (ex & dne).any() and (ex | dne).all()
    assert np.array_equal(ex, (labels != synth.ABSENT).T)
    assert pc[L + 4] == N and pc[L + 5] == 0
    # padding bits of the last word stay zero
    assert ((feas[:, -1] >> np.uint64(N % 64)) == 0).all()
    assert unk[4] == 2 and unk[L + 4] == 2 and (unk[np.r_[0:4, 5:L]] == 0).all()


@pytest.mark.parametrize("seed", [0, 1])
def test_inventory_flags_against_unique_values(orc, seed):
    """unknown bit 0 / bit 1 against numpy's unique values per label column."""
    wl = synth.affinity_workload(seed + 10, 400, 8, 300, card_choices=(3, 9, 30), absent_p=0.05)
    labels, row_off, term_off, preds = wl["labels"].copy(), wl["row_off"], wl["term_off"], wl["preds"]
    labels[:, 2] = synth.ABSENT
    labels[labels[:, 6] == 4, 6] = 5  # value 4 of label 6 disappears from the inventory
    _, _, unk, err = orc.affinity(labels, row_off, term_off, preds)
    assert err == 0
    carried = [set(np.unique(labels[:, l]).tolist()) - {synth.ABSENT} for l in range(labels.shape[1])]
    for i in range(row_off.shape[0] - 1):
        want = 0
        for t in range(row_off[i], row_off[i + 1]):
            for p in preds[term_off[t]:term_off[t + 1]]:
                l = int(p["label"])
                if not carried[l]:
                    want |= 2
                if int(p["op"]) in (0, 1):
                    vals = np.flatnonzero(np.unpackbits(p["vals"].view(np.uint8), bitorder="little"))
                    if any(int(v) not in carried[l] for v in vals):
                        want |= 1
        assert int(unk[i]) == want, i
    assert (unk & 1).any() and (unk & 2).any() and (unk == 0).any()


def test_malformed_affinity(orc):
    """Malformed expressions empty their term only; bad term offsets empty
    the term; bad row offsets empty the row; flags are input properties."""
    labels = np.array([[0, 1], [1, 1], [2, synth.ABSENT]], np.uint8)
    good = _pred(0, 0, [1, 2])  # nodes 1, 2
    rows = [
        [[good]],                                    # 0: nodes 1, 2
        [[_pred(0, 6)], [good]],                      # 1: op 6 -> term empty; row = nodes 1, 2
        [[_pred(2, 2)]],                              # 2: label >= L -> no node
        [[_pred(0, 4, thr=0)], [_pred(1, 2)]],        # 3: well-formed: node 1, 2 | node 0, 1
    ]
    row_off, term_off, preds = _csr(rows)
    feas, pc, unk, err = orc.affinity(labels, row_off, term_off, preds)
    assert err == 1  # F_PRED
    assert pc.tolist() == [2, 2, 0, 3]
    # Gt with vals[1] set, and value 255 in an In set, are malformed
    bad_gt = _pred(0, 4, thr=0)
    bad_gt["vals"][1] = 1
    bad_in = _pred(0, 0, [1])
    bad_in["vals"][3] |= np.uint64(1) << np.uint64(63)
    bad_rsv = good.copy()
    bad_rsv["rsv1"] = 1
    for bad in (bad_gt, bad_in, bad_rsv):
        row_off, term_off, preds = _csr([[[bad]], [[good]]])
        _, pc, unk, err = orc.affinity(labels, row_off, term_off, preds)
        assert err == 1 and pc.tolist() == [0, 2] and unk.tolist() == [0, 0]
    # a malformed expression in a term no row references still raises the flag
    row_off, term_off, preds = _csr([[[good]], [[bad_gt]]])
    _, pc, _, err = orc.affinity(labels, row_off[:2], term_off, preds)
    assert err == 1 and pc.tolist() == [2]
    # bad term offsets: that term is empty; bad row offsets: the row is empty
    row_off = np.array([0, 2, 1, 3], np.int32)
    term_off = np.array([0, 1, 9, 2], np.int32)  # term 1 = [1, 9) past n_preds = 2
    preds = np.array([good, _pred(1, 2)], synth.PRED_DT)
    feas, pc, unk, err = orc.affinity(labels, row_off, term_off, preds)
    assert err == 2  # F_OFFSETS
    assert pc.tolist() == [2, 0, 0]
