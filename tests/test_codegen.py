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
    assert len(ks) == 24   # 4 epilogues x 3 tile shapes x packed / one-run LoRA steps
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


def test_gelu_polynomial_error_bound():
    """The bf16 GELU epilogue's polynomial (coefficients read from the kernel
    header, evaluated in float32 in the kernel's order) stays within its
    stated error against the exact erf form: <= 1e-4 for |x| <= 4 and
    5.4e-5 |x| beyond (the fit error at the clamp point plus the normal tail)."""
    import numpy as np
    from scipy.special import erf
    src = open(os.path.join(CSRC, "vfm_internal.h")).read()
    body = src[src.index("__device__ inline float gelu_fast"):]
    body = body[:body.index("\n}\n")]
    lits = [float(v) for v in re.findall(r"(-?\d+\.\d*(?:e-?\d+)?)f", body)]
    assert len(lits) == 2 + 8 + 1, lits      # clamp +-4, the 8 coefficients, 0.5
    assert lits[0] == -4.0 and lits[1] == 4.0 and lits[-1] == 0.5
    coef = [np.float32(c) for c in lits[2:-1]]  # highest power first, as evaluated
    x = np.linspace(-12, 12, 2_400_001).astype(np.float32)
    t = np.clip(x, np.float32(-4), np.float32(4))
    u = t * t
    p = np.full_like(x, coef[0])
    for c in coef[1:]:
        p = (p * u + c).astype(np.float32)
    g = (x * (p * t + np.float32(0.5))).astype(np.float32)
    xd = x.astype(np.float64)
    ref = 0.5 * xd * (1.0 + erf(xd / np.sqrt(2.0)))
    err = np.abs(g - ref)
    inner = np.abs(x) <= 4
    assert err[inner].max() <= 1e-4, err[inner].max()
    assert np.all(err[~inner] <= 5.4e-5 * np.abs(xd[~inner]))
    # GELU(0) = 0 exactly, and odd symmetry of the polynomial part
    x0 = np.zeros(1, np.float32)
    p0 = np.full_like(x0, coef[0])
    for c in coef[1:]:
        p0 = (p0 * x0 * x0 + c).astype(np.float32)
    assert float((x0 * (p0 * x0 + np.float32(0.5)))[0]) == 0.0


def _regs(op):
    """Registers named by an operand: v5 -> {5}, v[4:7] -> {4..7} (VGPRs only)."""
    m = re.fullmatch(r"v(\d+)", op)
    if m:
        return {int(m.group(1))}
    m = re.fullmatch(r"v\[(\d+):(\d+)\]", op)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    return set()


def test_untracked_loads_not_touched_before_their_wait(all_asm):
    """Loads issued from inline asm are invisible to the compiler's wait
    insertion: the kernel's own s_waitcnt vmcnt must come before anything
    reads (or overwrites) their destination registers.  A register copy
    placed between such a load and its wait (for instance to carry the value
    around a loop) would read the register before the data landed.  The scan
    follows each kernel's instructions in program order, keeping the vector
    memory operations in flight; vmcnt(N) retires all but the last N."""
    vmem = re.compile(r"^(global_|buffer_|flat_|scratch_)")
    checked = 0
    for f, asm in all_asm.items():
        for name, body in _kernels(asm).items():
            inflight = []                                 # per VMEM op: its register set if untracked, else None
            in_asm = False
            for raw in body.splitlines():
                t = raw.strip()
                if t.startswith(";;#ASMSTART"):
                    in_asm = True
                    continue
                if t.startswith(";;#ASMEND"):
                    in_asm = False
                    continue
                l = t.split(";")[0].strip()
                if not l or l.endswith(":") or l.startswith("."):
                    continue
                mnem, _, rest = l.partition(" ")
                ops = [o.strip() for o in rest.split(",")] if rest else []
                if mnem == "s_waitcnt":
                    m = re.search(r"vmcnt\((\d+)\)", rest)
                    if m:
                        n = int(m.group(1))
                        inflight = inflight[len(inflight) - n:] if n else []
                    continue
                if not in_asm:
                    used = set().union(*(_regs(o) for o in ops)) if ops else set()
                    for regs in inflight:
                        if regs is not None:
                            assert not (used & regs), f"{f}: {name}: '{l}' touches an in-flight untracked load"
                if vmem.match(mnem):
                    if in_asm and mnem.startswith("global_load") and ops:
                        inflight.append(_regs(ops[0]))
                        checked += 1
                    else:
                        inflight.append(None)
    assert checked > 0
