"""pc_eval_selectors_noalloc, the selector entry point that allocates
nothing, against pc_eval_selectors: bit-exact bitsets, popcounts and
data-error flags on two calls in a row (the second smaller, so it runs on the
first call's leftovers in the fixed scratch), with the allocation hook set so
that any scratch growth would fail; a workload beyond the fixed maximum is
refused before any device work."""
import ctypes
import os

import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2602_16100_amd as pc
    return pc


def _p(t):
    return ctypes.c_void_p(t.data_ptr()) if t.numel() else None


def _noalloc(pc, ctx, wl, sentinel=0x33):
    """One call through the C ABI into sentinel-filled outputs; returns
    (rc, feasible, popcnt, flags)."""
    import torch
    N, L = wl["labels"].shape
    I = wl["pred_off"].shape[0] - 1
    W = (N + 63) // 64
    d = lambda a: pc.to_device(a, "cuda")  # noqa: E731
    labels, off, preds = d(wl["labels"]), d(wl["pred_off"]), d(wl["preds"])
    feas = torch.full((I, W), sentinel, dtype=torch.int64, device="cuda")
    pop = torch.full((I,), sentinel, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    ctx.data_errors(clear=True)
    rc = pc.lib().pc_eval_selectors_noalloc(ctx.handle, _p(labels), N, L, _p(off), _p(preds), preds.shape[0], I,
                                            _p(feas), _p(pop), None)
    torch.cuda.synchronize()
    flags = ctx.data_errors(clear=True)
    return rc, feas.cpu().numpy().view(np.uint64), pop.cpu().numpy().view(np.uint32), flags


def _reference(pc, ctx, wl):
    import torch
    d = lambda a: pc.to_device(a, "cuda")  # noqa: E731
    ctx.data_errors(clear=True)
    f, p = pc.pc_eval_selectors(d(wl["labels"]), d(wl["pred_off"]), d(wl["preds"]), ctx=ctx)
    torch.cuda.synchronize()
    flags = ctx.data_errors(clear=True)
    return f.cpu().numpy().view(np.uint64), p.cpu().numpy().view(np.uint32), flags


def _malformed(wl):
    """A few malformed predicates and offsets: the flags must agree too."""
    preds = wl["preds"].copy()
    preds[3]["label"] = 60000
    preds[7]["op"] = 9
    off = wl["pred_off"].copy()
    off[5], off[6] = off[6], off[5] - 1
    wl.arrays["preds"] = preds
    wl.arrays["pred_off"] = off
    return wl


def test_noalloc_matches_pc_eval_selectors(pc):
    ctx = pc.Context(0)
    big = _malformed(synth.selector_workload(31, 6000 + 17, 24, 3000, card_choices=(2, 4, 16, 64, 200),
                                             absent_p=0.05))
    small = synth.selector_workload(32, 700 + 5, 9, 120, absent_p=0.1)
    os.environ["PC_FAIL_ALLOC"] = "1"      # any scratch growth of the context would fail
    try:
        rc1, f1, p1, fl1 = _noalloc(pc, ctx, big)
        rc2, f2, p2, fl2 = _noalloc(pc, ctx, small)
    finally:
        del os.environ["PC_FAIL_ALLOC"]
    assert rc1 == pc.PC_OK, pc.lib().pc_last_error(ctx.handle)
    assert rc2 == pc.PC_OK, pc.lib().pc_last_error(ctx.handle)
    ref_ctx = pc.Context(0)
    rf1, rp1, rfl1 = _reference(pc, ref_ctx, big)
    rf2, rp2, rfl2 = _reference(pc, ref_ctx, small)
    assert np.array_equal(f1, rf1) and np.array_equal(p1, rp1) and fl1 == rfl1 and fl1 != 0
    assert np.array_equal(f2, rf2) and np.array_equal(p2, rp2) and fl2 == rfl2


def test_noalloc_refuses_beyond_its_maximum(pc):
    """Value planes of 64 labels x 256 values over 100,000 nodes need about
    200 MB: PC_EINVAL with the size, outputs untouched."""
    import torch
    ctx = pc.Context(0)
    wl = synth.selector_workload(33, 100000, 64, 10)
    rc, f, p, flags = _noalloc(pc, ctx, wl, sentinel=0x44)
    assert rc == pc.PC_EINVAL
    msg = pc.lib().pc_last_error(ctx.handle).decode()
    assert "pc_eval_selectors_noalloc" in msg and "bytes of scratch" in msg
    assert (f == np.uint64(0x44)).all() and (p == 0x44).all() and flags == 0
    # the context still serves the next call
    small = synth.selector_workload(34, 300, 5, 40)
    rc, f, p, flags = _noalloc(pc, ctx, small)
    rf, rp, rfl = _reference(pc, ctx, small)
    assert rc == pc.PC_OK and np.array_equal(f, rf) and np.array_equal(p, rp)
    torch.cuda.synchronize()
