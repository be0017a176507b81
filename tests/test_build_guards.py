"""Build guards for the flow-trace filter (CPU only: hipcc cross-compiles).

The match kernel's filter keeps each lane's chunk sets in registers that its
inline asm pins to v32..v127 and reads them in GPR index mode.  These tests
compile csrc/trace.hip for gfx950 and check, in the compiler's resource report
and in the kernel's own assembly, that this arrangement still holds under the
compiler at hand: no scratch (no spilled chunk sets) and at most 128 VGPRs (4
wavefronts per SIMD); every index-mode window is one of the filter blocks,
opened and closed inside it, holding only the indexed moves and ANDs that read
the pinned registers."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _hipcc():
    from paper_2602_16100_amd import _build
    cc = _build.hipcc()
    if not (os.path.exists(cc) or shutil.which(cc)):
        pytest.skip("hipcc not available")
    return cc, _build


@pytest.fixture(scope="module")
def match_build(tmp_path_factory):
    cc, B = _hipcc()
    out = tmp_path_factory.mktemp("guards")
    src = os.path.join(ROOT, "paper_2602_16100_amd", "csrc", "trace.hip")
    asm = str(out / "trace.s")
    r = subprocess.run([cc] + B.compile_flags() + ["--offload-device-only", "-S", src, "-o", asm,
                                                   "-Rpass-analysis=kernel-resource-usage"],
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-3000:]
    report = {}
    for block in r.stderr.split("remark: Function Name: ")[1:]:
        name = block.split()[0]
        vals = dict(re.findall(r"remark: \s*([A-Za-z ]+?)(?: \[[^\]]*\])?: (\d+)", block))
        report[name] = vals
    text = open(asm).read()
    m = re.search(r"^(_ZN\w*k_tr_match\w*):[^\n]*\n(.*?)^\s*s_endpgm", text, re.M | re.S)
    assert m, "k_tr_match not found in the assembly"
    return report, m.group(1), m.group(2)


def test_match_kernel_fits_without_spills(match_build):
    report, name, _ = match_build
    vals = report[name]
    assert int(vals["ScratchSize"]) == 0, vals
    assert int(vals.get("VGPRs Spill", 0)) == 0, vals
    assert int(vals["VGPRs"]) <= 128, vals
    assert int(vals["Occupancy"]) >= 4, vals


def test_index_mode_windows_are_the_filter_blocks(match_build):
    _, _, body = match_build
    lines = [ln.split(";")[0].strip() for ln in body.splitlines()]
    lines = [ln for ln in lines if ln and not ln.startswith((".", "//"))]
    windows, cur = [], None
    for ln in lines:
        op = ln.split()[0]
        if op == "s_set_gpr_idx_on":
            assert cur is None, "index mode opened twice"
            cur = []
        elif op == "s_set_gpr_idx_off":
            assert cur is not None, "index mode closed while off"
            windows.append(cur)
            cur = None
        elif cur is not None:
            cur.append(ln)
    assert cur is None, "index mode left on"
    assert len(windows) >= 2 and len(windows) % 2 == 0, len(windows)
    bases = set()
    for w in windows:
        assert len(w) == 23, w  # 12 indexed moves / ANDs and 11 index changes (4 lookups x 3 chunks)
        for ln in w:
            op = ln.split()[0]
            if op == "s_set_gpr_idx_idx":
                continue
            assert op in ("v_mov_b32", "v_and_b32", "v_mov_b32_e32", "v_and_b32_e32"), ln
            src = re.findall(r"\bv(\d+)\b", ln)
            # the indexed source is a chunk's first register, v32 + 16c
            assert any(int(v) in (32, 48, 64, 80, 96, 112) for v in src), ln
            bases.update(int(v) for v in src if int(v) in (32, 48, 64, 80, 96, 112))
    assert bases == {32, 48, 64, 80, 96, 112}
