"""Host-side checks of the C ABI (no GPU): the library loads and exports every
entry point declared in include/vfm.h; vfm_plan (host integer code) equals the
oracle's plan bit for bit; argument validation rejects bad calls before any
launch."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from oracle import vfm_oracle as O
from paper_2606_09643_amd import binding as B
from paper_2606_09643_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for f in os.listdir(os.path.join(ROOT, "include")):
        if f.endswith(".h"):
            src = open(os.path.join(ROOT, "include", f)).read()
            names |= set(re.findall(r"^\s*(?:int|const char\*)\s+(vfm_\w+)\s*\(", src, re.M))
    return names


def test_library_exports_every_declared_symbol():
    lib = B.lib()
    decl = _declared()
    assert {"vfm_plan", "vfm_layer_forward", "vfm_lora_apply", "vfm_head_forward"} <= decl
    for name in decl:
        assert hasattr(lib, name), name
    assert set(B.EXPORTS) == decl


def _unpack(host):
    n_req, n_tasks, T = int(host[0]), int(host[1]), int(host[2])
    p = B.VFM_PLAN_HEADER
    out = {}
    for name, n in [("order", n_req), ("task", n_req), ("cu_seqlens", n_req + 1),
                    ("seg_req", n_tasks + 1), ("seg_row", n_tasks + 1), ("cu_orig", n_req + 1),
                    ("logit_off", n_req + 1), ("ctx", n_req), ("kv_start", n_req),
                    ("qblk_off", n_req + 1), ("rtile_off", n_tasks + 1), ("row_task", T),
                    ("row_req", T), ("pos", T)]:
        out[name] = host[p:p + n].astype(np.int64)
        p += n
    assert p == host.size
    return out


@pytest.mark.parametrize("idx", [1, 2, 3, 4, 5])
def test_plan_matches_oracle_bit_exact(idx):
    w = wl.WORKLOADS[idx]
    b = wl.draw_batch(w)
    n_out = wl.draw_head_sizes(w)
    kvs = wl.kv_offsets(b).astype(np.int32) if b.ctx is not None else None
    host = B.vfm_plan(b.task_id, b.seq_len, w.n_tasks, b.ctx, kvs, n_out)
    got = _unpack(host)
    ref = O.plan(b.task_id, b.seq_len, w.n_tasks, ctx=b.ctx, n_out=n_out)
    for k in ("order", "task", "cu_seqlens", "seg_req", "seg_row", "cu_orig", "logit_off",
              "pos", "row_req"):
        assert np.array_equal(got[k], ref[k]), k
    assert np.array_equal(got["row_task"], ref["task"][ref["row_req"]])
    lens = b.seq_len[ref["order"]]
    assert np.array_equal(np.diff(got["qblk_off"]), (lens + 63) // 64)
    rows_t = np.diff(ref["seg_row"])
    assert np.array_equal(np.diff(got["rtile_off"]), (rows_t + 63) // 64)
    assert host[0] == w.n_req and host[1] == w.n_tasks and host[2] == b.total_rows
    assert host[3] == b.seq_len.max() and host[6] == ref["logit_off"][-1]


def test_plan_random_and_edges():
    r = np.random.default_rng(0)
    for _ in range(200):
        n_tasks = int(r.integers(1, 9))
        n_req = int(r.integers(1, 40))
        tid = r.integers(0, n_tasks, size=n_req)
        lens = r.integers(1, 300, size=n_req)
        host = B.vfm_plan(tid, lens, n_tasks)
        got, ref = _unpack(host), O.plan(tid, lens, n_tasks)
        for k in ("order", "cu_seqlens", "seg_req", "seg_row", "pos", "row_req"):
            assert np.array_equal(got[k], ref[k])


def test_plan_rejects_bad_input():
    with pytest.raises(B.VfmError) as e:
        B.vfm_plan([0, 4], [1, 1], 4)
    assert e.value.status == B.VFM_ERR_TASK
    with pytest.raises(B.VfmError) as e:
        B.vfm_plan([0, 1], [1, 0], 4)
    assert e.value.status == B.VFM_ERR_SHAPE
    with pytest.raises(B.VfmError):
        B.vfm_plan_size(0, 4, 0)


def _batch_c(host):
    return B.vfm_batch(host.ctypes.data_as(C.POINTER(C.c_int32)), 1 << 20, host.size)


def test_validation_rejects_before_launch():
    """Every call below fails host-side validation, so nothing reaches the GPU."""
    w = wl.WORKLOADS[2]
    host = B.vfm_plan([0, 1, 1], [5, 3, 2], 2)
    bc = _batch_c(host)
    lib = B.lib()
    cfg = B.make_cfg(B.VFM_BF16, 768, 12, 64, 3072, 0, 0, 0, 1, 1e-5, 0.0)
    n = C.c_size_t()
    assert lib.vfm_workspace_size(C.byref(cfg), C.byref(bc), None, C.byref(n)) == 0 and n.value > 0
    bad = B.make_cfg(B.VFM_BF16, 768, 8, 96, 3072, 0, 0, 0, 1, 1e-5, 0.0)
    assert lib.vfm_workspace_size(C.byref(bad), C.byref(bc), None, C.byref(n)) == B.VFM_ERR_UNSUPPORTED
    bad = B.make_cfg(B.VFM_BF16, 768, 11, 64, 3072, 0, 0, 0, 1, 1e-5, 0.0)
    assert lib.vfm_workspace_size(C.byref(bad), C.byref(bc), None, C.byref(n)) == B.VFM_ERR_SHAPE
    bad = B.make_cfg(7, 768, 12, 64, 3072, 0, 0, 0, 1, 1e-5, 0.0)
    assert lib.vfm_workspace_size(C.byref(bad), C.byref(bc), None, C.byref(n)) == B.VFM_ERR_ARG
    weights = B.vfm_layer_weights(*([1 << 20] * 13))
    x = 1 << 20
    # workspace missing
    st = lib.vfm_layer_forward(C.byref(cfg), C.byref(weights), None, C.byref(bc), x, None, None, 0,
                               None, 0, None)
    assert st == B.VFM_ERR_WORKSPACE
    # decode without a cache
    dec = B.make_cfg(B.VFM_BF16, 768, 12, 64, 3072, 0, 0, B.VFM_ATTN_DECODE, 1, 1e-5, 0.0)
    st = lib.vfm_layer_forward(C.byref(dec), C.byref(weights), None, C.byref(bc), x, None, None, 0,
                               1 << 20, 1 << 40, None)
    assert st == B.VFM_ERR_ARG
    # lora table for the wrong number of tasks
    lt = B.vfm_lora_table(5, 16, 1 << 20, 1 << 20)
    st = lib.vfm_layer_forward(C.byref(cfg), C.byref(weights), C.byref(lt), C.byref(bc), x, None,
                               None, 0, 1 << 20, 1 << 40, None)
    assert st == B.VFM_ERR_SHAPE
    # SwiGLU with biases is not supported
    sw = B.make_cfg(B.VFM_BF16, 768, 12, 64, 3072, 1, 1, 1, 1, 1e-6, 1e4)
    assert lib.vfm_workspace_size(C.byref(sw), C.byref(bc), None, C.byref(n)) == B.VFM_ERR_UNSUPPORTED
    assert B.vfm_status_string(B.VFM_ERR_TASK) == "task id out of range"


def test_binding_constants_match_header():
    """The binding's copies of the header's #define constants agree with it."""
    src = open(os.path.join(ROOT, "include", "vfm.h")).read()
    defs = dict(re.findall(r"#define\s+(VFM_\w+)\s+(\d+)", src))
    for name in ("VFM_PLAN_HEADER", "VFM_ROW_TILE", "VFM_SMALL_BATCH_ROWS"):
        assert int(defs[name]) == getattr(B, name), name
    mib = re.search(r"#define\s+VFM_NOALLOC_SCRATCH_BYTES\s+\(\(size_t\)(\d+) << 20\)", src)
    assert mib and int(mib.group(1)) << 20 == B.VFM_NOALLOC_SCRATCH_BYTES


def test_attach_rejects_bad_arguments_before_launching():
    """Argument errors of the runtime attach calls are found on the host (no
    GPU needed: nothing is launched when a check fails)."""
    lib = B.lib()
    fake = 0x10000                      # never dereferenced on these paths
    A = (B.C.c_void_p * B.VFM_NPROJ)()
    Bp = (B.C.c_void_p * B.VFM_NPROJ)()
    A[0] = fake
    Bp[0] = fake
    tab = B.vfm_lora_table(4, 16, fake, fake, (B.C.c_void_p * B.VFM_NPROJ)(fake, 0, 0, 0, 0, 0, 0),
                           (B.C.c_void_p * B.VFM_NPROJ)(fake, 0, 0, 0, 0, 0, 0))
    at = lambda t, r, a=A, b=Bp: lib.vfm_lora_attach(B.C.byref(tab), t, r, 1.0, B.C.cast(a, B.C.c_void_p),
                                                     B.C.cast(b, B.C.c_void_p), None)
    assert at(4, 8) == B.VFM_ERR_TASK
    assert at(-1, 8) == B.VFM_ERR_TASK
    assert at(0, 12) == B.VFM_ERR_SHAPE          # not a multiple of 8
    assert at(0, 24) == B.VFM_ERR_SHAPE          # above max_rank
    A2 = (B.C.c_void_p * B.VFM_NPROJ)(fake, fake, 0, 0, 0, 0, 0)
    B2 = (B.C.c_void_p * B.VFM_NPROJ)(fake, fake, 0, 0, 0, 0, 0)
    assert at(0, 8, A2, B2) == B.VFM_ERR_ARG     # projection 1 has no table array
    B3 = (B.C.c_void_p * B.VFM_NPROJ)(0, 0, 0, 0, 0, 0, 0)
    assert at(0, 8, A, B3) == B.VFM_ERR_ARG      # A without B
    assert lib.vfm_lora_attach(None, 0, 0, 0.0, None, None, None) == B.VFM_ERR_ARG
    ht = B.vfm_head_table(4, B.VFM_POOL_MEAN, 10, fake, fake, 0, 0, 0, None, None)
    ha = lambda t, n, W, b, W1=None, b1=None: lib.vfm_head_attach(B.C.byref(ht), t, n, W, b, W1, b1, None)
    assert ha(4, 5, fake, None) == B.VFM_ERR_TASK
    assert ha(0, 11, fake, None) == B.VFM_ERR_SHAPE
    assert ha(0, 5, None, None) == B.VFM_ERR_ARG
    assert ha(0, 5, fake, fake) == B.VFM_ERR_ARG          # no bias array
    assert ha(0, 5, fake, None, fake) == B.VFM_ERR_ARG    # MLP layer without MLP tables


def test_encoder_calls_reject_bad_arguments_before_launching():
    """vfm_embed_series / vfm_encoder_attach argument errors are found on the
    host (nothing is launched when a check fails)."""
    lib = B.lib()
    fake = 0x10000
    host = B.vfm_plan([0, 1, 1], [5, 3, 2], 2)
    bc = _batch_c(host)
    cfg = B.make_cfg(B.VFM_BF16, 1024, 16, 64, 2816, 0, 0, 0, 1, 1e-5, 0.0)
    emb = lambda enc, patch=8, src=fake, W=fake, x=fake: lib.vfm_embed_series(
        C.byref(cfg), C.byref(bc), enc, src, patch, W, None, x, None)
    good = B.vfm_encoder_table(2, 3, fake, None)
    assert emb(None) == B.VFM_ERR_ARG
    assert emb(C.byref(good), src=None) == B.VFM_ERR_ARG
    assert emb(C.byref(good), W=None) == B.VFM_ERR_ARG
    assert emb(C.byref(B.vfm_encoder_table(2, 3, None, None))) == B.VFM_ERR_ARG
    assert emb(C.byref(B.vfm_encoder_table(3, 3, fake, None))) == B.VFM_ERR_SHAPE   # task count
    assert emb(C.byref(B.vfm_encoder_table(2, 0, fake, None))) == B.VFM_ERR_SHAPE
    assert emb(C.byref(B.vfm_encoder_table(2, 65, fake, None))) == B.VFM_ERR_SHAPE
    assert emb(C.byref(good), patch=0) == B.VFM_ERR_SHAPE
    assert emb(C.byref(good), patch=65) == B.VFM_ERR_SHAPE
    att = lambda tab, t, W=fake, b=None: lib.vfm_encoder_attach(tab, t, W, b, None)
    assert att(C.byref(good), 2) == B.VFM_ERR_TASK
    assert att(C.byref(good), -1) == B.VFM_ERR_TASK
    assert att(C.byref(good), 0, fake, fake) == B.VFM_ERR_ARG                        # no bias array
    assert att(None, 0) == B.VFM_ERR_ARG


def test_paged_layer_rejects_bad_pages_before_launch():
    """vfm_layer_forward_paged validates the page size, the page table
    against the pool and the step kind on the host (nothing is launched when
    a check fails)."""
    lib = B.lib()
    fake = 1 << 20
    # two decode tokens (ctx 40 and 10) and, for the mixed cases, a prompt
    host = B.vfm_plan([0, 1], [1, 1], 2, [40, 10], None)
    bc = _batch_c(host)
    cfg = B.make_cfg(B.VFM_BF16, 4096, 32, 128, 11008, 1, 1, B.VFM_ATTN_DECODE, 0, 1e-6, 1e4)
    weights = B.vfm_layer_weights(*([fake] * 13))
    table = np.array([[3, 1, 2], [0, 0, 0]], np.int32)       # request 0 needs 3 pages of 16, request 1 one

    def run(tab=table, page=16, n_pages=4, c=cfg, batch=bc, k=fake):
        kv = B.vfm_kv_pages(k, fake, n_pages, page, tab.shape[1],
                            tab.ctypes.data_as(C.POINTER(C.c_int32)), fake)
        return lib.vfm_layer_forward_paged(C.byref(c), C.byref(weights), None, C.byref(batch), fake,
                                           C.byref(kv), fake, 1 << 40, None)
    assert run(k=None) == B.VFM_ERR_ARG
    assert run(page=24) == B.VFM_ERR_ARG                       # not a power of two
    assert run(page=8) == B.VFM_ERR_ARG                        # below 16
    assert run(n_pages=3) == B.VFM_ERR_SHAPE                   # page 3 is outside the pool
    assert run(tab=np.array([[3, 1], [0, 0]], np.int32)) == B.VFM_ERR_SHAPE   # 41 tokens need 3 pages
    assert run(tab=np.array([[3, 1, -1], [0, 0, 0]], np.int32)) == B.VFM_ERR_SHAPE
    bidir = B.make_cfg(B.VFM_BF16, 4096, 32, 128, 11008, 1, 1, B.VFM_ATTN_BIDIR, 0, 1e-6, 1e4)
    assert run(c=bidir) == B.VFM_ERR_UNSUPPORTED
    # mixed steps: a request with cached tokens and more than one new row is a prompt chunk
    mixed32 = B.make_cfg(B.VFM_F32, 4096, 32, 128, 11008, 1, 1, B.VFM_ATTN_MIXED, 0, 1e-6, 1e4)
    chunked = B.vfm_plan([0, 1], [2, 1], 2, [40, 0], None)
    assert run(c=mixed32, batch=_batch_c(chunked)) == B.VFM_ERR_UNSUPPORTED   # prompt chunks: bf16 only
    decode_many = B.vfm_plan([0, 1], [1, 5], 2, [0, 0], None)
    assert run(batch=_batch_c(decode_many)) == B.VFM_ERR_UNSUPPORTED   # decode rows are single


def test_prompt_steps_refuse_cached_context():
    """Bidirectional and causal steps attend over a request's own rows only,
    so a request that brings cached tokens (ctx > 0) is refused on the host
    (contiguous and paged entry points alike) instead of ignoring them; the
    same batch is accepted as a mixed step."""
    lib = B.lib()
    fake = 1 << 20
    weights = B.vfm_layer_weights(*([fake] * 13))
    host = B.vfm_plan([0, 1], [3, 2], 2, [0, 17], None)        # request 1: a chunk after 17 tokens
    bc = _batch_c(host)
    zero = _batch_c(B.vfm_plan([0, 1], [3, 2], 2, [0, 0], None))
    table = np.array([[0], [1]], np.int32)

    def cfg(attn):
        return B.make_cfg(B.VFM_BF16, 4096, 32, 128, 11008, 1, 1, attn, 0, 1e-6, 1e4)

    def plain(c, batch, kc=fake):
        return lib.vfm_layer_forward(C.byref(c), C.byref(weights), None, C.byref(batch), fake,
                                     kc, kc, 1 << 20, fake, 1 << 40, None)

    def paged(c, batch):
        kv = B.vfm_kv_pages(fake, fake, 4, 64, 1, table.ctypes.data_as(C.POINTER(C.c_int32)), fake)
        return lib.vfm_layer_forward_paged(C.byref(c), C.byref(weights), None, C.byref(batch), fake,
                                           C.byref(kv), fake, 1 << 40, None)

    for attn in (B.VFM_ATTN_BIDIR, B.VFM_ATTN_CAUSAL):
        assert plain(cfg(attn), bc) == B.VFM_ERR_UNSUPPORTED
        assert plain(cfg(attn), bc, kc=None) == B.VFM_ERR_UNSUPPORTED
    assert paged(cfg(B.VFM_ATTN_CAUSAL), bc) == B.VFM_ERR_UNSUPPORTED
    # without cached tokens the same shapes pass this check and stop at the
    # workspace check that follows it (a null workspace; nothing launched)
    c = cfg(B.VFM_ATTN_CAUSAL)
    assert lib.vfm_layer_forward(C.byref(c), C.byref(weights), None, C.byref(zero), fake,
                                 None, None, 0, None, 0, None) == B.VFM_ERR_WORKSPACE


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one GPU only: --gpus above 1 exits with status 2
    and says so, before touching a device."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    p = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "4"], cwd=root,
                       capture_output=True, text=True, timeout=300)
    assert p.returncode == 2, (p.returncode, p.stdout[-500:], p.stderr[-500:])
    assert "one GPU only" in p.stdout + p.stderr
