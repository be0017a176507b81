"""The issue-rate microbenchmark behind the instruction-issue rooflines
(pc_measure_valu): two-source 32-bit VALU operations on vector registers
retire about twice as fast as three-source ones, the scalar unit about as
fast as the latter, and the shader clock it reads under load is a plausible
MI355X clock.  Bad arguments return PC_EINVAL without launching anything."""
import ctypes

import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2602_16100_amd as pc
    return pc


def test_issue_classes_and_clock(pc):
    ctx = pc.Context(0)
    full, clk = ctx.measure_valu(0, 3)    # v_add_u32 / v_sub_u32
    half, _ = ctx.measure_valu(2, 3)      # v_and_or_b32, three vector sources
    salu, _ = ctx.measure_valu(6, 3)      # s_xor_b32
    assert 1.0e9 < clk < 3.0e9, clk
    assert full > 0 and half > 0 and salu > 0
    # the two VALU classes differ by about 2x (measured 1.86 / 0.98 per CU per clock)
    assert 1.6 < full / half < 2.4, (full, half)
    assert 0.7 < salu / half < 1.3, (salu, half)


def test_bad_arguments(pc):
    ctx = pc.Context(0)
    L = pc.lib()
    r, c = ctypes.c_double(-1.0), ctypes.c_double(-1.0)
    for op, reps in ((-1, 1), (15, 1), (0, 0)):
        assert L.pc_measure_valu(ctx.handle, op, reps, ctypes.byref(r), ctypes.byref(c), None) == pc.PC_EINVAL
    assert L.pc_measure_valu(ctx.handle, 0, 1, None, ctypes.byref(c), None) == pc.PC_EINVAL
    assert r.value == -1.0 and c.value == -1.0
