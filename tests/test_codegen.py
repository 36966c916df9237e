"""Properties of the compiled gfx950 code that the kernels' speed depends on
and that a source change can silently lose (CPU only: hipcc cross-compiles
each source to assembly with the library's own flags).

- No kernel uses private (scratch) memory or spills vector registers (SGPR
  spills go to VGPR lanes, not memory, and are allowed), except the fp32
  G = 8 attention, which keeps its per-chunk row table (indexed by a runtime
  chunk number) in scratch beside 250 VGPRs of accumulators: it is the
  reference-precision route, not the bf16 decode path.
- The fused selection with whole blocks per wave issues all sixteen of a
  thread's index-row requests (eight 16-byte code loads and eight 8-byte
  parameter loads) before its first wait on any of them, so the rows of the
  eight candidate slots are in flight together.
"""
import concurrent.futures
import glob
import importlib.util
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2604_07815_amd", "csrc")


def _build_module():
    spec = importlib.util.spec_from_file_location("tls_build", os.path.join(ROOT, "paper_2604_07815_amd", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.fixture(scope="module")
def assembly(tmp_path_factory):
    b = _build_module()
    if not shutil.which(b.HIPCC) and not os.path.exists(b.HIPCC):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("asm")

    def compile_one(src):
        dst = os.path.join(out, os.path.basename(src) + ".s")
        r = subprocess.run([b.HIPCC, *b.CFLAGS, "--cuda-device-only", "-S", src, "-o", dst], capture_output=True,
                           text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        return os.path.basename(src), open(dst).read()

    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        return dict(ex.map(compile_one, srcs))


def _kernel_metadata(asm):
    """(name, private segment bytes, VGPR spills, SGPR spills) of every kernel."""
    out = []
    for blk in asm.split("  - .agpr_count")[1:]:
        name = re.search(r"\.name:\s+(\S+)", blk).group(1)
        field = lambda k: int(re.search(r"\." + k + r":\s+(\d+)", blk).group(1))
        out.append((name, field("private_segment_fixed_size"), field("vgpr_spill_count"), field("sgpr_spill_count")))
    return out


SCRATCH_ALLOWED = {"_ZN3tls15attn_gqa_kernelINS_3F32ELi128ELi8EEEvPKNT_1TES5_S5_PKilNS_9TokenListES7_iiiiiiifPfS9_Pj"}


def test_no_kernel_uses_scratch_or_spills(assembly):
    seen = 0
    for src, asm in assembly.items():
        for name, priv, vsp, ssp in _kernel_metadata(asm):
            seen += 1
            if name in SCRATCH_ALLOWED:
                continue
            assert priv == 0 and vsp == 0, (src, name, priv, vsp)
    assert seen >= 40


def test_fused_selection_rows_in_flight_together(assembly):
    asm = assembly["token_select_mfma.hip"]
    bodies = re.findall(r"^(_ZN3tls24token_select_mfma_kernelILi\dELb1E\S*):[^\n]*\n(.*?)s_endpgm", asm, flags=re.S | re.M)
    assert len(bodies) == 4  # G = 1..4
    for name, body in bodies:
        lines = body.splitlines()
        first = next(i for i, l in enumerate(lines) if re.search(r"global_load_dwordx4 .* nt$", l.strip()))
        issued = 0
        for l in lines[first:]:
            t = l.strip()
            if re.match(r"global_load_dwordx[24] .* nt$", t):
                issued += 1
            elif t.startswith("s_waitcnt") and "vmcnt" in t:
                break
        assert issued == 16, (name, issued)
