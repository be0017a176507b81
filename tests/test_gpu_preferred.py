"""Parity of pc_score_preferred (through the C ABI) with the CPU oracle:
best node, score, tie count and the data-error word, bit-exact, on seeded
clusters spanning several 8,192-node tiles with ragged tails, with and
without a feasible bitset, every operator, programs long enough to exhaust
the compiled-program buffer (rows decoded on the fly), malformed inputs,
the paper's 5-worker fixture, and sampled rows at the combined workload's
full size."""
import json
import os

import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu
HERE = os.path.dirname(os.path.abspath(__file__))
OPS = {"In": 0, "NotIn": 1, "Exists": 2, "DoesNotExist": 3, "Gt": 4, "Lt": 5}


@pytest.fixture(scope="module")
def g():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import gpu_run
    return gpu_run


def _same(a, b, what):
    a, b = np.asarray(a), np.asarray(b)
    assert a.shape == b.shape, (what, a.shape, b.shape)
    bad = np.argwhere(a != b)
    assert bad.size == 0, f"{what}: first mismatch at {tuple(bad[0])}: gpu {a[tuple(bad[0])]} oracle {b[tuple(bad[0])]}"


def _pack(bits):
    I, N = bits.shape
    W = (N + 63) // 64
    pad = np.zeros((I, W * 64), np.uint8)
    pad[:, :N] = bits
    return np.packbits(pad, axis=1, bitorder="little").view(np.uint64).reshape(I, W)


def _check(g, orc, labels, row_off, term_off, weight, preds, feasible=None, n_terms=None, n_preds=None, rows=None):
    bg, sg, cg, eg = g.preferred(labels, row_off, term_off, weight, preds, feasible=feasible, n_terms=n_terms,
                                 n_preds=n_preds)
    bo, so, co, eo = orc.preferred(labels, row_off, term_off, weight, preds, feasible=feasible, n_terms=n_terms,
                                   n_preds=n_preds, rows=rows)
    if rows is not None:
        bg, sg, cg = bg[rows], sg[rows], cg[rows]
    _same(bg, bo, "best")
    _same(sg, so, "score")
    _same(cg, co, "count")
    assert eg == eo, (eg, eo)
    return bo, so, co


@pytest.mark.parametrize("seed,N,absent,p_feas", [(0, 5037, 0.1, 0.3), (1, 20000 + 5, 0.0, None),
                                                  (2, 100, 0.3, 0.5), (3, 64 * 781 - 40, 0.05, 0.02)])
def test_preferred_random(g, orc, seed, N, absent, p_feas):
    wl = synth.affinity_workload(seed, N, 12, 1, card_choices=(2, 3, 16, 64, 200), absent_p=absent)
    row_off, term_off, preds, weight = synth.preferred_rows(seed, wl.meta["cards"], 700, tmin=0, tmax=6, kmin=0,
                                                            kmax=4)
    feas = None if p_feas is None else _pack(np.random.default_rng(seed).random((700, N)) < p_feas)
    bo, so, co = _check(g, orc, wl["labels"], row_off, term_off, weight, preds, feasible=feas)
    assert (so > 0).sum() > 100 and (co > 1).sum() > 10


def test_preferred_plane_tables_past_2gib(g, orc):
    """8,000 labels over 3,000 nodes: the plane tables pass 2 GiB, so the
    evaluator reads them through 64-bit pointers."""
    wl = synth.affinity_workload(43, 3000, 8000, 1, card_choices=(2, 3, 16, 64), absent_p=0.05)
    row_off, term_off, preds, weight = synth.preferred_rows(43, wl.meta["cards"], 300, tmin=0, tmax=6, kmin=0, kmax=4)
    bo, so, co = _check(g, orc, wl["labels"], row_off, term_off, weight, preds)
    assert (so > 0).sum() > 50


@pytest.mark.parametrize("seed,wmax", [(5, 1), (6, 2), (7, 3)])
def test_preferred_few_terms_ties(g, orc, seed, wmax):
    """Rows of zero to three terms (the term-pattern class) with weights of
    at most wmax, so that different patterns of holding terms share a score
    and the best nodes come from several patterns at once; with and without
    a feasible bitset, several tiles and a ragged tail."""
    N = 3 * 8192 + 77
    wl = synth.affinity_workload(seed, N, 10, 1, card_choices=(2, 3, 5), absent_p=0.1)
    row_off, term_off, preds, weight = synth.preferred_rows(seed, wl.meta["cards"], 900, tmin=0, tmax=3, kmin=1,
                                                            kmax=2)
    weight = (weight % wmax + 1).astype(np.uint32)
    for feas in (None, _pack(np.random.default_rng(seed).random((900, N)) < 0.4)):
        bo, so, co = _check(g, orc, wl["labels"], row_off, term_off, weight, preds, feasible=feas)
        assert (co > 1).sum() > 100


def test_preferred_paper_fixture(g, orc):
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
    row_off, term_off, preds, weight, feas = [0], [0], [], [], []
    for case in fx["cases"]:
        for w, term in case["terms"]:
            for k, op, vals in term:
                p = np.zeros(1, synth.PRED_DT)[0]
                p["label"], p["op"] = keys.index(k), OPS[op]
                bm = [0, 0, 0, 0]
                for v in vals:
                    c = codes[k][v]
                    bm[c >> 6] |= 1 << (c & 63)
                p["vals"] = np.array(bm, np.uint64)
                preds.append(p)
            term_off.append(len(preds))
            weight.append(w)
        row_off.append(len(term_off) - 1)
        feas.append([True] * len(nodes) if case["feasible"] is None else [nm in case["feasible"] for nm in names])
    bo, so, co = _check(g, orc, labels, np.array(row_off, np.int32), np.array(term_off, np.int32),
                        np.array(weight, np.uint32), np.array(preds, synth.PRED_DT), feasible=_pack(np.array(feas)))
    for r, case in enumerate(fx["cases"]):
        want = -1 if case["best"] is None else names.index(case["best"])
        assert (int(bo[r]), int(so[r]), int(co[r])) == (want, case["score"], case["count"]), case["cite"]


def test_preferred_long_programs_decode(g, orc):
    """In / NotIn sets of up to 120 values on 250-value labels: programs far
    beyond 4 entries per expression exhaust the compiled-program buffer, so
    most rows are decoded on the fly; the rest run from the buffer."""
    rng = np.random.default_rng(5)
    N, L = 9000 + 3, 4
    cards = np.array([250, 250, 7, 3])
    labels = synth.gen_labels(rng, N, cards, absent_p=0.05)
    I = 300
    row_off, term_off, preds, weight = [0], [0], [], []
    for i in range(I):
        for t in range(int(rng.integers(1, 5))):
            for e in range(int(rng.integers(1, 3))):
                p = np.zeros(1, synth.PRED_DT)[0]
                lab = int(rng.integers(0, L))
                p["label"], p["op"] = lab, int(rng.integers(0, 2))
                vals = rng.choice(cards[lab], size=int(rng.integers(1, min(120, cards[lab]) + 1)), replace=False)
                bm = [0, 0, 0, 0]
                for v in vals:
                    bm[int(v) >> 6] |= 1 << (int(v) & 63)
                p["vals"] = np.array(bm, np.uint64)
                preds.append(p)
            term_off.append(len(preds))
            weight.append(int(rng.integers(1, 101)))
        row_off.append(len(term_off) - 1)
    _check(g, orc, labels, np.array(row_off, np.int32), np.array(term_off, np.int32), np.array(weight, np.uint32),
           np.array(preds, synth.PRED_DT), feasible=_pack(rng.random((I, N)) < 0.6))


def test_preferred_malformed(g, orc):
    wl = synth.affinity_workload(8, 3000, 6, 1, card_choices=(2, 4, 16))
    row_off, term_off, preds, weight = synth.preferred_rows(8, wl.meta["cards"], 200)
    weight = weight.copy()
    weight[3], weight[10] = 0, 101
    preds = preds.copy()
    preds[5]["label"] = 60          # label >= L
    preds[9]["op"] = 7              # bad operator
    term_off = term_off.copy()
    term_off[20] = term_off[21] + 1  # a bad term offset pair (terms 19 and 20)
    row_off = row_off.copy()
    row_off[50] = row_off[51] + 2    # a bad row offset pair (rows 49 and 50)
    _check(g, orc, wl["labels"], row_off, term_off, weight, preds)
    # a row of 656 terms (malformed) and one of 655 (fine)
    good = preds[:1]
    big_preds = np.repeat(good, 656 + 655)
    t_off = np.arange(656 + 655 + 1, dtype=np.int32)
    _check(g, orc, wl["labels"], np.array([0, 656, 656 + 655], np.int32), t_off,
           np.full(656 + 655, 100, np.uint32), big_preds)


def test_preferred_empty(g, orc):
    wl = synth.affinity_workload(9, 500, 4, 1, card_choices=(2, 4))
    row_off, term_off, preds, weight = synth.preferred_rows(9, wl.meta["cards"], 30, tmin=0, tmax=2)
    # no rows; no nodes; no terms anywhere; an all-zero feasible bitset
    _check(g, orc, wl["labels"], row_off[:1], term_off, weight, preds)
    _check(g, orc, np.zeros((0, 4), np.uint8), row_off, term_off, weight, preds)
    _check(g, orc, wl["labels"], np.zeros(31, np.int32), np.zeros(1, np.int32), np.zeros(0, np.uint32),
           np.zeros(0, synth.PRED_DT))
    _check(g, orc, wl["labels"], row_off, term_off, weight, preds, feasible=np.zeros((30, 8), np.uint64))


def test_preferred_full_size_sampled(g, orc):
    """The combined workload's cluster (50,000 nodes x 64 labels) and 699,051
    preferred rows, every row on the GPU; 600 sampled rows against the
    oracle, with a seeded random feasible bitset (about half the nodes)."""
    wl = synth.affinity_workload(4, 50000, 64, 1)
    I = 699051
    row_off, term_off, preds, weight = synth.preferred_rows(4, wl.meta["cards"], I)
    feas = np.random.default_rng(44).integers(0, 2 ** 64 - 1, size=(I, 782), dtype=np.uint64, endpoint=True)
    rows = np.sort(np.random.default_rng(46).choice(I, size=600, replace=False)).astype(np.int32)
    rows = np.concatenate([rows, np.array([0, I - 1], np.int32)])
    bo, so, co = _check(g, orc, wl["labels"], row_off, term_off, weight, preds, feasible=feas, rows=rows)
    assert (so > 0).sum() > 300
