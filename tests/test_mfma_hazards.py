"""gfx950 assembly of the MFMA kernels: no MFMA result is read by a vector
instruction before it is ready, on any path (CPU only: hipcc cross-compiles)."""
import concurrent.futures as cf
import os
import subprocess

import pytest

from mfma_hazards import early_reads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2407_15462_amd", "csrc")
SOURCES = ["mol_fused.hip", "mol_rerank.hip", "mol_pairwise.hip", "mol_per_embd.hip", "mol_dots.hip"]
HIPCC = "/opt/rocm/bin/hipcc"


def _asm(src: str, tmp: str) -> str:
    out = os.path.join(tmp, src + ".s")
    cmd = [HIPCC, "-O3", "-std=c++17", "--offload-arch=gfx950", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "--cuda-device-only", "-S",
           os.path.join(CSRC, src), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return open(out).read()


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_no_mfma_result_read_early(tmp_path):
    with cf.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        listings = dict(zip(SOURCES, ex.map(lambda s: _asm(s, str(tmp_path)), SOURCES)))
    bad = {s: early_reads(a, need=8) for s, a in listings.items()}
    bad = {s: v for s, v in bad.items() if v}
    assert not bad, "\n".join(f"{s}: {x}" for s, v in bad.items() for x in v[:5])


def test_checker_flags_a_read_across_a_skipped_block():
    # a result read right after a branch that skips the padding block
    asm = "\n".join([
        "_Zk:",
        "\tv_mfma_f32_16x16x32_f16 v[2:5], v[10:13], v[14:17], v[2:5]",
        "\ts_cbranch_scc1 .LBB0_2",
        "\ts_nop 7",
        "\ts_nop 7",
        ".LBB0_2:",
        "\tv_exp_f32_e32 v0, v3",
        "\ts_endpgm",
        ".Lfunc_end0:",
    ])
    assert len(early_reads(asm, need=8)) == 1
    # with the padding before the branch the read is safe
    safe = asm.replace("\ts_cbranch_scc1", "\ts_nop 7\n\ts_cbranch_scc1")
    assert early_reads(safe, need=8) == []
