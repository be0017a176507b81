"""Pins of the CPU oracle's preferred node affinity (per row: the feasible
node of largest summed weight of holding terms, the lowest index among
equals; its score and the number of feasible nodes that reach it).

The preference oracle is checked against things it does not compute itself:
- the paper's 5-worker label matrix with hand-derived winners, scores and
  tie counts (golden fixture);
- a decomposition through the separately pinned required-affinity oracle:
  every preferred term evaluated as a one-term required row, the weighted
  sum and the first maximum taken with numpy;
- invariants: scaling every weight scales every score and keeps the winner,
  permuting a row's terms or adding a term that holds nowhere changes
  nothing, no feasibility input equals an all-ones bitset;
- closed forms for empty rows, empty feasible sets and malformed inputs.
"""
import json
import os

import numpy as np
import pytest

import synth

HERE = os.path.dirname(os.path.abspath(__file__))
OPS = {"In": 0, "NotIn": 1, "Exists": 2, "DoesNotExist": 3, "Gt": 4, "Lt": 5}
F_PRED, F_OFFSETS = 1, 2


def _pred(label, op, vals=()):
    p = np.zeros(1, synth.PRED_DT)[0]
    p["label"] = label
    p["op"] = op
    bm = [0, 0, 0, 0]
    for v in vals:
        bm[int(v) >> 6] |= 1 << (int(v) & 63)
    p["vals"] = np.array(bm, np.uint64)
    return p


def _csr(rows):
    """rows: list of rows, a row a list of (weight, [preds])."""
    row_off, term_off, preds, weight = [0], [0], [], []
    for row in rows:
        for w, term in row:
            preds.extend(term)
            term_off.append(len(preds))
            weight.append(w)
        row_off.append(len(term_off) - 1)
    arr = np.array(preds, synth.PRED_DT) if preds else np.zeros(0, synth.PRED_DT)
    return (np.array(row_off, np.int32), np.array(term_off, np.int32), arr, np.array(weight, np.uint32))


def _pack(bits):
    """bool [I, N] -> u64 [I, W]"""
    I, N = bits.shape
    W = (N + 63) // 64
    pad = np.zeros((I, W * 64), np.uint8)
    pad[:, :N] = bits
    return np.packbits(pad, axis=1, bitorder="little").view(np.uint64).reshape(I, W)


def _unpack(feas, N):
    return np.unpackbits(feas.view(np.uint8), bitorder="little", axis=-1)[..., :N].astype(bool)


def test_paper_label_matrix_preferences(orc):
    fx = json.load(open(os.path.join(HERE, "golden", "paper_preferred.json")))
    keys, nodes = fx["keys"], fx["nodes"]
    names = [n["name"] for n in nodes]
    codes = {k: {v: i for i, v in enumerate(sorted({n[k] for n in nodes if k in n}))} for k in keys}
    for case in fx["cases"]:
        for _, term in case["terms"]:
            for k, _, vals in term:
                for v in vals:
                    codes[k].setdefault(v, len(codes[k]))
    labels = np.full((len(nodes), len(keys)), synth.ABSENT, np.uint8)
    for i, n in enumerate(nodes):
        for j, k in enumerate(keys):
            if k in n:
                labels[i, j] = codes[k][n[k]]
    rows, feas = [], np.zeros((len(fx["cases"]), len(nodes)), bool)
    for r, case in enumerate(fx["cases"]):
        rows.append([(w, [_pred(keys.index(k), OPS[op], [codes[k][v] for v in vals]) for k, op, vals in term])
                     for w, term in case["terms"]])
        feas[r] = True if case["feasible"] is None else [nm in case["feasible"] for nm in names]
    row_off, term_off, preds, weight = _csr(rows)
    best, score, count, err = orc.preferred(labels, row_off, term_off, weight, preds, feasible=_pack(feas))
    assert err == 0
    for r, case in enumerate(fx["cases"]):
        want = -1 if case["best"] is None else names.index(case["best"])
        assert (int(best[r]), int(score[r]), int(count[r])) == (want, case["score"], case["count"]), case["cite"]


def _by_decomposition(orc, labels, row_off, term_off, preds, weight, feas_bits):
    """Scores from one-term required-affinity rows, summed with numpy."""
    T = term_off.shape[0] - 1
    N = labels.shape[0]
    one = np.arange(T + 1, dtype=np.int32)  # row t = term t alone
    f, _, _, _ = orc.affinity(labels, one, term_off, preds)
    holds = _unpack(f, N)  # [T, N]
    w_ok = np.where((weight >= 1) & (weight <= 100), weight, 0).astype(np.int64)
    I = row_off.shape[0] - 1
    best = np.full(I, -1, np.int32)
    score = np.zeros(I, np.uint32)
    count = np.zeros(I, np.uint32)
    for i in range(I):
        tb, te = int(row_off[i]), int(row_off[i + 1])
        sc = (w_ok[tb:te, None] * holds[tb:te]).sum(axis=0) if te > tb else np.zeros(N, np.int64)
        m = feas_bits[i]
        if not m.any():
            continue
        top = sc[m].max()
        best[i] = int(np.flatnonzero(m & (sc == top))[0])
        score[i] = top
        count[i] = int((m & (sc == top)).sum())
    return best, score, count


@pytest.mark.parametrize("seed,N,absent,p_feas", [(0, 300, 0.1, 0.5), (1, 1000 + 7, 0.0, 0.9), (2, 64, 0.3, 0.05)])
def test_preferences_match_term_decomposition(orc, seed, N, absent, p_feas):
    wl = synth.affinity_workload(seed, N, 9, 1, card_choices=(2, 3, 16, 64, 200), absent_p=absent)
    labels = wl["labels"]
    row_off, term_off, preds, weight = synth.preferred_rows(seed, wl.meta["cards"], 400, tmin=0, tmax=5, kmin=0,
                                                            kmax=3)
    rng = np.random.default_rng(seed)
    feas_bits = rng.random((400, N)) < p_feas
    feas_bits[:5] = False  # rows without a feasible node
    best, score, count, err = orc.preferred(labels, row_off, term_off, weight, preds, feasible=_pack(feas_bits))
    assert err == 0
    b2, s2, c2 = _by_decomposition(orc, labels, row_off, term_off, preds, weight, feas_bits)
    assert np.array_equal(best, b2) and np.array_equal(score, s2) and np.array_equal(count, c2)
    assert (best[:5] == -1).all() and (score[:5] == 0).all() and (count[:5] == 0).all()
    assert np.array_equal(count >= 1, feas_bits.any(axis=1)) and np.array_equal(best >= 0, feas_bits.any(axis=1))
    assert (score > 0).sum() > 50  # the workload exercises real scores


def test_invariants(orc):
    wl = synth.affinity_workload(4, 500, 8, 1, card_choices=(2, 4, 16, 64))
    labels = wl["labels"]
    row_off, term_off, preds, weight = synth.preferred_rows(4, wl.meta["cards"], 300, tmin=1, tmax=4)
    small = (weight % 10 + 1).astype(np.uint32)  # 1..10
    b1, s1, c1, _ = orc.preferred(labels, row_off, term_off, small, preds)
    # scaling every weight by 10 scales every score and keeps winners and tie counts
    b2, s2, c2, _ = orc.preferred(labels, row_off, term_off, small * 10, preds)
    assert np.array_equal(b1, b2) and np.array_equal(s2, s1 * 10) and np.array_equal(c1, c2)
    # no feasibility input = every node feasible
    allf = np.full((300, (500 + 63) // 64), ~np.uint64(0), np.uint64)
    b3, s3, c3, _ = orc.preferred(labels, row_off, term_off, small, preds, feasible=allf)
    assert np.array_equal(b1, b3) and np.array_equal(s1, s3) and np.array_equal(c1, c3)
    # reversing the terms of every row changes nothing
    perm = np.concatenate([np.arange(row_off[i + 1] - 1, row_off[i] - 1, -1) for i in range(300)]).astype(np.int64)
    lens = np.diff(term_off)[perm]
    t_off2 = np.zeros(perm.shape[0] + 1, np.int32)
    t_off2[1:] = np.cumsum(lens)
    preds2 = np.concatenate([preds[term_off[t]:term_off[t + 1]] for t in perm]) if preds.size else preds
    b4, s4, c4, _ = orc.preferred(labels, row_off, t_off2, small[perm], preds2)
    assert np.array_equal(b1, b4) and np.array_equal(s1, s4) and np.array_equal(c1, c4)
    # a term that holds nowhere (DoesNotExist of a label every node carries), weight 100, in every row
    rows_new, preds_new, w_new, t_new = [0], [], [], [0]
    for i in range(300):
        for t in range(row_off[i], row_off[i + 1]):
            preds_new.extend(preds[term_off[t]:term_off[t + 1]])
            t_new.append(len(preds_new))
            w_new.append(small[t])
        preds_new.append(_pred(0, OPS["DoesNotExist"]))
        t_new.append(len(preds_new))
        w_new.append(100)
        rows_new.append(len(t_new) - 1)
    b5, s5, c5, _ = orc.preferred(labels, np.array(rows_new, np.int32), np.array(t_new, np.int32),
                                  np.array(w_new, np.uint32), np.array(preds_new, synth.PRED_DT))
    assert np.array_equal(b1, b5) and np.array_equal(s1, s5) and np.array_equal(c1, c5)


def test_row_subset_reads_each_rows_own_feasible_bits(orc):
    """rows= evaluates the listed rows only, each against its own row of the
    feasible bitset."""
    wl = synth.affinity_workload(6, 200, 6, 1, card_choices=(2, 4, 16))
    row_off, term_off, preds, weight = synth.preferred_rows(6, wl.meta["cards"], 50)
    feas_bits = np.random.default_rng(6).random((50, 200)) < 0.3
    fb = _pack(feas_bits)
    full = orc.preferred(wl["labels"], row_off, term_off, weight, preds, feasible=fb)
    sub = np.array([49, 3, 17, 3, 0], np.int32)
    part = orc.preferred(wl["labels"], row_off, term_off, weight, preds, feasible=fb, rows=sub)
    for a, b in zip(full[:3], part[:3]):
        assert np.array_equal(a[sub], b)


def test_empty_and_malformed(orc):
    labels = np.array([[0, 1], [1, 1], [2, 0], [1, 255]], np.uint8)
    good = [_pred(0, OPS["In"], [1])]  # nodes 1 and 3
    # a row with no terms: first feasible node, score 0, all tie
    ro, to, pr, w = _csr([[]])
    assert orc.preferred(labels, ro, to, w, pr)[:3] == (np.array([0]), np.array([0]), np.array([4]))
    # weight 0 and 101: the term counts for no node, PRED raised
    for bad in (0, 101):
        ro, to, pr, w = _csr([[(bad, good), (3, [_pred(1, OPS["In"], [0])])]])
        b, s, c, err = orc.preferred(labels, ro, to, w, pr)
        assert (int(b[0]), int(s[0]), int(c[0]), err) == (2, 3, 1, F_PRED)
    # a malformed expression (label out of range) empties its term only
    ro, to, pr, w = _csr([[(50, [_pred(7, OPS["Exists"])]), (9, good)]])
    b, s, c, err = orc.preferred(labels, ro, to, w, pr)
    assert (int(b[0]), int(s[0]), int(c[0]), err) == (1, 9, 2, F_PRED)
    # a bad term offset pair: the term holds nowhere, OFFSETS raised
    ro, to, pr, w = _csr([[(9, good), (5, good)]])
    to2 = to.copy()
    to2[2] = 0  # term 1 = [1, 0): reversed
    b, s, c, err = orc.preferred(labels, ro, to2, w, pr)
    assert (int(b[0]), int(s[0]), int(c[0]), err) == (1, 9, 2, F_OFFSETS)
    # a row of 656 terms is malformed: no terms (score 0 everywhere), OFFSETS raised; 655 terms are fine
    for n_t, want in ((655, (1, 655, 2, 0)), (656, (0, 0, 4, F_OFFSETS))):
        ro, to, pr, w = _csr([[(1, good)] * n_t])
        b, s, c, err = orc.preferred(labels, ro, to, w, pr)
        assert (int(b[0]), int(s[0]), int(c[0]), err) == want
    # no feasible node
    ro, to, pr, w = _csr([[(9, good)]])
    b, s, c, err = orc.preferred(labels, ro, to, w, pr, feasible=np.zeros((1, 1), np.uint64))
    assert (int(b[0]), int(s[0]), int(c[0])) == (-1, 0, 0)
    # padding bits past N in the feasible bitset are ignored
    b, s, c, err = orc.preferred(labels, ro, to, w, pr, feasible=np.array([[np.uint64(0xF0)]], np.uint64))
    assert (int(b[0]), int(s[0]), int(c[0])) == (-1, 0, 0)
