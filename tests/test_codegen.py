"""Code-generation checks of the gfx950 kernels (CPU only: hipcc
cross-compiles to AMD assembly).

* No kernel spills to scratch.
* In the large-tile GEMM, the global->LDS loads of the next K step stay in
  flight while the current step's fragments are read: no `s_waitcnt vmcnt`
  immediately before a `ds_read_b128` (the compiler inserts one whenever it
  cannot tell the two LDS stages apart, which serialises load and compute).
* No packed fp32 arithmetic is emitted.
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_09643_amd", "csrc")

pytestmark = pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                                reason="hipcc not available")


def _asm(src):
    from paper_2606_09643_amd.build import FLAGS, _hipcc
    out = subprocess.run([_hipcc(), *FLAGS, "--cuda-device-only", "-S", os.path.join(CSRC, src), "-o", "-"],
                         capture_output=True, text=True)
    assert out.returncode == 0, out.stderr[-2000:]
    return out.stdout


def _kernels(asm):
    """{kernel symbol: body text}"""
    res = {}
    for m in re.finditer(r"^(_Z\S+):\s*(?:;.*)?$", asm, re.M):
        name = m.group(1)
        end = asm.find("s_endpgm", m.end())
        res[name] = asm[m.end():end]
    return res


@pytest.fixture(scope="module")
def all_asm():
    return {f: _asm(f) for f in sorted(os.listdir(CSRC)) if f.endswith(".hip")}


def test_no_scratch_spills(all_asm):
    for f, asm in all_asm.items():
        for name, size in re.findall(r"\.set (\S+)\.private_seg_size, (\d+)", asm):
            assert int(size) == 0, f"{f}: {name} uses {size} bytes of scratch"


def test_large_gemm_keeps_lds_dma_in_flight(all_asm):
    ks = {k: v for k, v in _kernels(all_asm["k_gemm.hip"]).items() if "gemm_bf16_large_kernel" in k}
    assert len(ks) == 12   # 4 epilogues x 3 tile shapes
    for name, body in ks.items():
        lines = [l.strip() for l in body.splitlines() if l.strip() and not l.strip().startswith(";")]
        assert any(l.startswith("global_load_lds_dwordx4") for l in lines), name
        for prev, cur in zip(lines, lines[1:]):
            if cur.startswith("ds_read_b128"):
                assert "vmcnt" not in prev, f"{name}: DMA wait before a fragment read"


def test_no_packed_fp32(all_asm):
    for f, asm in all_asm.items():
        assert not re.search(r"\bv_pk_(add|mul|fma)_f32\b", asm), f


def test_lds_reads_stay_lds(all_asm):
    """LDS tiles are read with ds_* instructions: a pointer into LDS that the
    compiler loses track of (e.g. passed through an asm statement) becomes a
    generic pointer and every fragment read turns into a flat load through the
    vector-memory pipeline."""
    for f in ("k_attn.hip", "k_decode.hip", "k_segmented.hip", "k_rows.hip"):
        for name, body in _kernels(all_asm[f]).items():
            assert not re.search(r"^\s+flat_(load|store)", body, re.M), f"{f}: {name} uses flat memory ops"
    for name, body in _kernels(all_asm["k_gemm.hip"]).items():
        if "gemm_bf16_large_kernel" in name:
            assert not re.search(r"^\s+flat_(load|store)", body, re.M), name
