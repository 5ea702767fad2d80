"""ctypes binding of ``libvfm.so`` (declared in ``include/vfm.h``).

Argument marshalling only: every step of the forward runs inside the HIP
library.  PyTorch provides device memory and the stream.  The functions keep
the C names (``vfm_plan``, ``vfm_layer_forward``, ...); the small classes
below build the C structs (plan buffers, per-task pointer tables) from torch
tensors and keep those tensors alive while the structs are in use.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np
import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libvfm.so")

VFM_OK, VFM_ERR_ARG, VFM_ERR_SHAPE, VFM_ERR_TASK = 0, -1, -2, -3
VFM_ERR_UNSUPPORTED, VFM_ERR_WORKSPACE, VFM_ERR_HIP = -4, -5, -6
VFM_F32, VFM_BF16 = 0, 1
VFM_NORM_LAYER, VFM_NORM_RMS = 0, 1
VFM_MLP_GELU, VFM_MLP_SWIGLU = 0, 1
VFM_ATTN_BIDIR, VFM_ATTN_CAUSAL, VFM_ATTN_DECODE, VFM_ATTN_MIXED = 0, 1, 2, 3
VFM_POOL_MEAN, VFM_POOL_FIRST, VFM_POOL_LAST = 0, 1, 2
VFM_EMBED_ROWS, VFM_EMBED_TOKENS, VFM_EMBED_PATCHES = 0, 1, 2
VFM_ACT_GELU, VFM_ACT_RELU = 0, 1
VFM_NPROJ = 7
VFM_PLAN_HEADER = 16
VFM_ROW_TILE = 64
VFM_SMALL_BATCH_ROWS = 1024
VFM_NOALLOC_SCRATCH_BYTES = 128 << 20
PROJ = ("q", "k", "v", "o", "gate", "up", "down")

EXPORTS = ("vfm_status_string", "vfm_plan_size", "vfm_plan", "vfm_workspace_size",
           "vfm_embed_forward", "vfm_layer_forward", "vfm_lora_apply", "vfm_head_forward",
           "vfm_profile_enable", "vfm_profile_read",
           "vfm_bfq_state_size", "vfm_bfq_init", "vfm_bfq_enqueue", "vfm_bfq_next_batch",
           "vfm_bfq_queued", "vfm_bfq_tags", "vfm_lora_attach", "vfm_head_attach",
           "vfm_embed_series", "vfm_encoder_attach", "vfm_layer_forward_paged", "vfm_greedy_tokens",
           "vfm_pages_state_size", "vfm_pages_init", "vfm_pages_reserve", "vfm_pages_release",
           "vfm_pages_table", "vfm_pages_count", "vfm_bfq_charge",
           "vfm_layer_forward_noalloc")
PROF_CLASSES = ("gemm_qkv", "gemm_o", "gemm_up", "gemm_down", "attn", "norm", "shrink", "other")


class VfmError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {_lib_handle().vfm_status_string(status).decode()} ({status})")


class vfm_cfg(C.Structure):
    _fields_ = [("dtype", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("head_dim", C.c_int32), ("d_ff", C.c_int32), ("norm", C.c_int32),
                ("mlp", C.c_int32), ("attn", C.c_int32), ("has_bias", C.c_int32),
                ("norm_eps", C.c_float), ("rope_theta", C.c_float)]


class vfm_batch(C.Structure):
    _fields_ = [("plan_host", C.POINTER(C.c_int32)), ("plan_dev", C.c_void_p),
                ("n_ints", C.c_size_t)]


class vfm_layer_weights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("norm1_w", "norm1_b", "w_qkv", "b_qkv", "w_o", "b_o",
                                           "norm2_w", "norm2_b", "w_gate", "w_up", "b_up",
                                           "w_down", "b_down")]


class vfm_lora_table(C.Structure):
    _fields_ = [("n_tasks", C.c_int32), ("max_rank", C.c_int32), ("rank", C.c_void_p),
                ("scale", C.c_void_p), ("A", C.c_void_p * VFM_NPROJ), ("B", C.c_void_p * VFM_NPROJ)]


class vfm_head_table(C.Structure):
    _fields_ = [("n_tasks", C.c_int32), ("pool", C.c_int32), ("max_out", C.c_int32),
                ("n_out", C.c_void_p), ("W", C.c_void_p), ("b", C.c_void_p),
                ("hidden", C.c_int32), ("act", C.c_int32), ("W1", C.c_void_p), ("b1", C.c_void_p)]


class vfm_kv_pages(C.Structure):
    _fields_ = [("k", C.c_void_p), ("v", C.c_void_p), ("n_pages", C.c_int64), ("page_size", C.c_int32),
                ("max_pages", C.c_int32), ("table_host", C.POINTER(C.c_int32)), ("table_dev", C.c_void_p)]


class vfm_pages_config(C.Structure):
    _fields_ = [("n_pages", C.c_int32), ("page_size", C.c_int32), ("max_seqs", C.c_int32),
                ("max_pages", C.c_int32)]


_LIB = None


def _lib_handle():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"HIP library {LIB_PATH} is not built; run "
                               "`python -m paper_2606_09643_amd.build` (no CPU fallback exists)")
        lib = C.CDLL(LIB_PATH)
        lib.vfm_status_string.restype = C.c_char_p
        lib.vfm_status_string.argtypes = [C.c_int]
        lib.vfm_plan_size.argtypes = [C.c_int32, C.c_int32, C.c_int64, C.POINTER(C.c_size_t)]
        lib.vfm_plan.argtypes = [C.c_void_p] * 5 + [C.c_int32, C.c_int32, C.c_void_p, C.c_size_t]
        lib.vfm_workspace_size.argtypes = [C.POINTER(vfm_cfg), C.POINTER(vfm_batch),
                                           C.POINTER(vfm_lora_table), C.POINTER(C.c_size_t)]
        lib.vfm_embed_forward.argtypes = [C.POINTER(vfm_cfg), C.POINTER(vfm_batch), C.c_int32,
                                          C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p,
                                          C.c_void_p, C.c_void_p]
        lib.vfm_layer_forward.argtypes = [C.POINTER(vfm_cfg), C.POINTER(vfm_layer_weights),
                                          C.POINTER(vfm_lora_table), C.POINTER(vfm_batch),
                                          C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64,
                                          C.c_void_p, C.c_size_t, C.c_void_p]
        lib.vfm_layer_forward_noalloc.argtypes = [C.POINTER(vfm_cfg), C.POINTER(vfm_layer_weights),
                                                  C.POINTER(vfm_lora_table), C.POINTER(vfm_batch),
                                                  C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64, C.c_void_p]
        lib.vfm_layer_forward_paged.argtypes = [C.POINTER(vfm_cfg), C.POINTER(vfm_layer_weights),
                                                C.POINTER(vfm_lora_table), C.POINTER(vfm_batch), C.c_void_p,
                                                C.POINTER(vfm_kv_pages), C.c_void_p, C.c_size_t, C.c_void_p]
        lib.vfm_greedy_tokens.argtypes = [C.POINTER(vfm_batch), C.c_void_p, C.c_void_p, C.c_void_p]
        lib.vfm_pages_state_size.argtypes = [C.POINTER(vfm_pages_config), C.POINTER(C.c_size_t)]
        lib.vfm_pages_init.argtypes = [C.POINTER(vfm_pages_config), C.c_void_p, C.c_size_t]
        lib.vfm_pages_reserve.argtypes = [C.c_void_p, C.c_int32, C.c_int64]
        lib.vfm_pages_release.argtypes = [C.c_void_p, C.c_int32]
        lib.vfm_pages_table.argtypes = [C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_int32]
        lib.vfm_pages_count.argtypes = [C.c_void_p, C.c_int32, C.POINTER(C.c_int32), C.POINTER(C.c_int32)]
        lib.vfm_lora_apply.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                       C.POINTER(vfm_lora_table), C.POINTER(vfm_batch),
                                       C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]
        lib.vfm_head_forward.argtypes = [C.POINTER(vfm_cfg), C.c_void_p, C.c_void_p,
                                         C.POINTER(vfm_head_table), C.POINTER(vfm_batch),
                                         C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t,
                                         C.c_void_p]
        lib.vfm_profile_enable.argtypes = [C.c_uint32]
        lib.vfm_profile_read.argtypes = [C.c_void_p, C.c_void_p, C.c_int32]
        lib.vfm_lora_attach.argtypes = [C.POINTER(vfm_lora_table), C.c_int32, C.c_int32, C.c_float,
                                        C.c_void_p, C.c_void_p, C.c_void_p]
        lib.vfm_head_attach.argtypes = [C.POINTER(vfm_head_table), C.c_int32, C.c_int32, C.c_void_p,
                                        C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        lib.vfm_embed_series.argtypes = [C.POINTER(vfm_cfg), C.POINTER(vfm_batch),
                                         C.POINTER(vfm_encoder_table), C.c_void_p, C.c_int32,
                                         C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        lib.vfm_encoder_attach.argtypes = [C.POINTER(vfm_encoder_table), C.c_int32, C.c_void_p,
                                           C.c_void_p, C.c_void_p]
        lib.vfm_bfq_state_size.argtypes = [C.POINTER(vfm_bfq_config), C.POINTER(C.c_size_t)]
        lib.vfm_bfq_init.argtypes = [C.POINTER(vfm_bfq_config), C.c_void_p, C.c_size_t]
        lib.vfm_bfq_enqueue.argtypes = [C.c_void_p, C.c_int32, C.c_int64, C.c_double, C.c_double]
        lib.vfm_bfq_next_batch.argtypes = [C.c_void_p, C.c_double, C.c_void_p, C.c_void_p, C.c_int32,
                                           C.POINTER(C.c_int32)]
        lib.vfm_bfq_charge.argtypes = [C.c_void_p, C.c_int32, C.c_double]
        lib.vfm_bfq_queued.argtypes = [C.c_void_p, C.c_int32, C.POINTER(C.c_int32)]
        lib.vfm_bfq_tags.argtypes = [C.c_void_p, C.c_int32, C.c_int32, C.POINTER(C.c_double),
                                     C.POINTER(C.c_double)]
        for name in EXPORTS:
            getattr(lib, name).restype = C.c_int if name != "vfm_status_string" else C.c_char_p
        _LIB = lib
    return _LIB


def lib():
    """The loaded library (raises if it was not built)."""
    return _lib_handle()


def _check(st: int, where: str):
    if st != VFM_OK:
        raise VfmError(st, where)


def _ptr(t) -> int | None:
    if t is None:
        return None
    if isinstance(t, torch.Tensor):
        return t.data_ptr()
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return int(t)


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


# --------------------------------------------------------------------------
# C entry points
# --------------------------------------------------------------------------
def vfm_status_string(status: int) -> str:
    return _lib_handle().vfm_status_string(status).decode()


def vfm_plan_size(n_req: int, n_tasks: int, total_rows: int) -> int:
    n = C.c_size_t()
    _check(_lib_handle().vfm_plan_size(n_req, n_tasks, total_rows, C.byref(n)), "vfm_plan_size")
    return n.value


def vfm_plan(task_id, seq_len, n_tasks, ctx_len=None, kv_start=None, n_out=None) -> np.ndarray:
    """Host plan buffer (int32) for a batch; see include/vfm.h for its layout."""
    a = lambda v: None if v is None else np.ascontiguousarray(v, dtype=np.int32)
    task_id, seq_len, ctx_len, kv_start, n_out = map(a, (task_id, seq_len, ctx_len, kv_start, n_out))
    n_req = int(task_id.shape[0])
    n = vfm_plan_size(n_req, n_tasks, int(seq_len.astype(np.int64).sum()))
    out = np.zeros(n, np.int32)
    st = _lib_handle().vfm_plan(_ptr(task_id), _ptr(seq_len), _ptr(ctx_len), _ptr(kv_start),
                                _ptr(n_out), n_req, n_tasks, _ptr(out), n)
    _check(st, "vfm_plan")
    return out


def vfm_workspace_size(cfg: vfm_cfg, batch: vfm_batch, lora: vfm_lora_table | None = None) -> int:
    n = C.c_size_t()
    st = _lib_handle().vfm_workspace_size(C.byref(cfg), C.byref(batch),
                                          C.byref(lora) if lora is not None else None, C.byref(n))
    _check(st, "vfm_workspace_size")
    return n.value


def vfm_embed_forward(cfg, batch, mode, src, src_width, table, bias, x, stream=None):
    st = _lib_handle().vfm_embed_forward(C.byref(cfg), C.byref(batch), mode, _ptr(src), src_width,
                                         _ptr(table), _ptr(bias), _ptr(x), _stream(stream))
    _check(st, "vfm_embed_forward")


def vfm_layer_forward(cfg, weights, lora, batch, x, k_cache=None, v_cache=None, kv_slots=0,
                      workspace=None, stream=None):
    ws_ptr, ws_bytes = (workspace.data_ptr(), workspace.numel() * workspace.element_size()) \
        if workspace is not None else (None, 0)
    st = _lib_handle().vfm_layer_forward(C.byref(cfg), C.byref(weights),
                                         C.byref(lora) if lora is not None else None,
                                         C.byref(batch), _ptr(x), _ptr(k_cache), _ptr(v_cache),
                                         kv_slots, ws_ptr, ws_bytes, _stream(stream))
    _check(st, "vfm_layer_forward")


def vfm_layer_forward_noalloc(cfg, weights, lora, batch, x, k_cache=None, v_cache=None, kv_slots=0,
                              stream=None):
    st = _lib_handle().vfm_layer_forward_noalloc(C.byref(cfg), C.byref(weights),
                                                 C.byref(lora) if lora is not None else None,
                                                 C.byref(batch), _ptr(x), _ptr(k_cache), _ptr(v_cache),
                                                 kv_slots, _stream(stream))
    _check(st, "vfm_layer_forward_noalloc")


class PagedKV:
    """One layer's paged K / V pool (device tensors [n_heads, n_pages * page_size,
    head_dim]) with a page table (host int32 [n_req, max_pages], original
    request order) and its device copy, as the C struct vfm_kv_pages."""

    def __init__(self, k, v, page_size, table, device="cuda"):
        self.k, self.v = k, v
        self.table = np.ascontiguousarray(table, np.int32)
        self.table_dev = torch.from_numpy(self.table).to(device)
        self.c = vfm_kv_pages(k.data_ptr(), v.data_ptr(), k.shape[1] // page_size, int(page_size),
                              self.table.shape[1], self.table.ctypes.data_as(C.POINTER(C.c_int32)),
                              self.table_dev.data_ptr())


def vfm_layer_forward_paged(cfg, weights, lora, batch, x, kv, workspace, stream=None):
    """kv: a PagedKV, or a vfm_kv_pages struct built by the caller."""
    kvc = kv.c if isinstance(kv, PagedKV) else kv
    st = _lib_handle().vfm_layer_forward_paged(C.byref(cfg), C.byref(weights),
                                               C.byref(lora) if lora is not None else None,
                                               C.byref(batch), _ptr(x), C.byref(kvc), workspace.data_ptr(),
                                               workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "vfm_layer_forward_paged")


def vfm_lora_apply(dtype, proj, d_in, d_out, lora, batch, x, y, workspace, stream=None):
    st = _lib_handle().vfm_lora_apply(dtype, proj, d_in, d_out, C.byref(lora), C.byref(batch),
                                      _ptr(x), _ptr(y), workspace.data_ptr(),
                                      workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "vfm_lora_apply")


def vfm_head_forward(cfg, final_norm_w, final_norm_b, heads, batch, x, out, workspace, stream=None):
    ws_ptr, ws_bytes = (workspace.data_ptr(), workspace.numel() * workspace.element_size()) \
        if workspace is not None else (None, 0)
    st = _lib_handle().vfm_head_forward(C.byref(cfg), _ptr(final_norm_w), _ptr(final_norm_b),
                                        C.byref(heads) if heads is not None else None,
                                        C.byref(batch), _ptr(x), _ptr(out), ws_ptr, ws_bytes,
                                        _stream(stream))
    _check(st, "vfm_head_forward")


def vfm_profile_enable(classes=()) -> None:
    """Bracket launches of the named kernel classes with hipEvents (0 = off)."""
    mask = 0
    for c in classes:
        mask |= 1 << PROF_CLASSES.index(c)
    _check(_lib_handle().vfm_profile_enable(mask), "vfm_profile_enable")


def vfm_profile_read() -> dict:
    """{class: (total_ms, launches)} since the last vfm_profile_enable."""
    n = len(PROF_CLASSES)
    ms = np.zeros(n, np.float64)
    cnt = np.zeros(n, np.int64)
    _check(_lib_handle().vfm_profile_read(ms.ctypes.data, cnt.ctypes.data, n), "vfm_profile_read")
    return {c: (float(ms[i]), int(cnt[i])) for i, c in enumerate(PROF_CLASSES)}


# --------------------------------------------------------------------------
# struct builders (keep the tensors they point to alive)
# --------------------------------------------------------------------------
def make_cfg(dtype, d_model, n_heads, head_dim, d_ff, norm, mlp, attn, has_bias, norm_eps,
             rope_theta) -> vfm_cfg:
    return vfm_cfg(dtype, d_model, n_heads, head_dim, d_ff, norm, mlp, attn, int(has_bias),
                   norm_eps, rope_theta)


class Batch:
    """A planned batch: host plan, its device copy and the C struct."""

    def __init__(self, task_id, seq_len, n_tasks, ctx_len=None, kv_start=None, n_out=None,
                 device="cuda", non_blocking=False):
        self.host = vfm_plan(task_id, seq_len, n_tasks, ctx_len, kv_start, n_out)
        if non_blocking:     # staged through pinned memory: the host does not wait for the stream
            self.dev = torch.from_numpy(self.host).pin_memory().to(device, non_blocking=True)
        else:
            self.dev = torch.from_numpy(self.host).to(device)
        self.c = vfm_batch(self.host.ctypes.data_as(C.POINTER(C.c_int32)), self.dev.data_ptr(),
                           self.host.size)

    @property
    def n_req(self):
        return int(self.host[0])

    @property
    def T(self):
        return int(self.host[2])

    @property
    def total_outputs(self):
        return int(self.host[6])

    def out_off(self):
        """out_off[n_req + 1] of the host plan: first head output of request i (original order)."""
        n, t = self.n_req, int(self.host[1])
        o = VFM_PLAN_HEADER + n + n + (n + 1) + (t + 1) + (t + 1) + (n + 1)
        return self.host[o:o + n + 1]


def layer_weights(W: dict) -> vfm_layer_weights:
    return vfm_layer_weights(*[_ptr(W.get(n)) for n, _ in vfm_layer_weights._fields_])


class LoraTable:
    """Device pointer tables of per-task LoRA factors for one layer.

    factors: {proj: (list of A_t tensors or None, list of B_t tensors or None)}.
    """

    def __init__(self, n_tasks, ranks, scales, factors: dict, max_rank=None, device="cuda"):
        ranks = np.asarray(ranks, np.int32)
        self.rank = torch.from_numpy(ranks).to(device)
        self.scale = torch.as_tensor(np.asarray(scales, np.float32)).to(device)
        mr = int(ranks.max()) if max_rank is None else int(max_rank)
        self._keep = []
        A = (C.c_void_p * VFM_NPROJ)()
        B = (C.c_void_p * VFM_NPROJ)()
        for p, name in enumerate(PROJ):
            if name not in factors:
                continue
            As, Bs = factors[name]
            pa = torch.tensor([_ptr(a) if a is not None and a.numel() else 0 for a in As],
                              dtype=torch.int64).to(device)
            pb = torch.tensor([_ptr(b) if b is not None and b.numel() else 0 for b in Bs],
                              dtype=torch.int64).to(device)
            self._keep += [pa, pb, As, Bs]
            A[p] = pa.data_ptr()
            B[p] = pb.data_ptr()
        self.c = vfm_lora_table(n_tasks, mr, self.rank.data_ptr(), self.scale.data_ptr(), A, B)


def vfm_lora_attach(table, task, rank, scale, A=None, B=None, stream=None):
    """Rewrites task `task`'s adapter entries of a LoRA table (rank 0 removes
    them).  A, B: {proj name: device tensor} of the task's factors."""
    a = (C.c_void_p * VFM_NPROJ)()
    b = (C.c_void_p * VFM_NPROJ)()
    for p, name in enumerate(PROJ):
        if A is not None and name in A:
            a[p] = _ptr(A[name])
            b[p] = _ptr(B[name])
    st = _lib_handle().vfm_lora_attach(C.byref(table.c), int(task), int(rank), float(scale),
                                       C.cast(a, C.c_void_p), C.cast(b, C.c_void_p), _stream(stream))
    _check(st, "vfm_lora_attach")


def vfm_head_attach(table, task, n_out, W=None, b=None, W1=None, b1=None, stream=None):
    st = _lib_handle().vfm_head_attach(C.byref(table.c), int(task), int(n_out), _ptr(W), _ptr(b),
                                       _ptr(W1), _ptr(b1), _stream(stream))
    _check(st, "vfm_head_attach")


class HeadTable:
    """Device tables of per-task heads.  W1s / b1s (optional): per task the
    MLP head's first layer [hidden, d] / [hidden] (None = linear head)."""

    def __init__(self, n_out, Ws, bs, pool, device="cuda", W1s=None, b1s=None, hidden=0,
                 act=VFM_ACT_GELU):
        n_out = np.asarray(n_out, np.int32)
        self.n_out = torch.from_numpy(n_out).to(device)
        self._keep = [Ws, bs, W1s, b1s]
        ptrs = lambda xs: torch.tensor([_ptr(x) if x is not None else 0 for x in xs],
                                       dtype=torch.int64).to(device)
        self.pw, self.pb = ptrs(Ws), ptrs(bs)
        self.pw1 = ptrs(W1s) if W1s is not None else None
        self.pb1 = ptrs(b1s) if b1s is not None else None
        self.c = vfm_head_table(len(n_out), pool, int(n_out.max()) if n_out.size else 0,
                                self.n_out.data_ptr(), self.pw.data_ptr(), self.pb.data_ptr(),
                                int(hidden), int(act),
                                self.pw1.data_ptr() if self.pw1 is not None else None,
                                self.pb1.data_ptr() if self.pb1 is not None else None)


class vfm_encoder_table(C.Structure):
    _fields_ = [("n_tasks", C.c_int32), ("n_channels", C.c_int32), ("W", C.c_void_p), ("b", C.c_void_p)]


class EncoderTable:
    """Device tables of per-task channel-combiner encoders: Ws[t] float32 [C]
    or None (no encoder: channel 0 passes), bs[t] float32 [1] or None."""

    def __init__(self, n_channels, Ws, bs=None, device="cuda"):
        self._keep = [Ws, bs]
        ptrs = lambda xs: torch.tensor([_ptr(x) if x is not None else 0 for x in xs],
                                       dtype=torch.int64).to(device)
        self.pw = ptrs(Ws)
        self.pb = ptrs(bs) if bs is not None else None
        self.c = vfm_encoder_table(len(Ws), int(n_channels), self.pw.data_ptr(),
                                   self.pb.data_ptr() if self.pb is not None else None)


def vfm_embed_series(cfg, batch, enc, src, patch, W_pe, b_pe, x, stream=None):
    st = _lib_handle().vfm_embed_series(C.byref(cfg), C.byref(batch), C.byref(enc.c), _ptr(src), int(patch),
                                        _ptr(W_pe), _ptr(b_pe), _ptr(x), _stream(stream))
    _check(st, "vfm_embed_series")


def vfm_encoder_attach(enc, task, W=None, b=None, stream=None):
    st = _lib_handle().vfm_encoder_attach(C.byref(enc.c), int(task), _ptr(W), _ptr(b), _stream(stream))
    _check(st, "vfm_encoder_attach")


def vfm_greedy_tokens(batch, out, ids, stream=None):
    _check(_lib_handle().vfm_greedy_tokens(C.byref(batch), _ptr(out), _ptr(ids), _stream(stream)),
           "vfm_greedy_tokens")


# ---- KV page allocator (host, include/vfm_pages.h) --------------------------
class PageAllocator:
    """The library's page allocator on a host state buffer (numpy-owned)."""

    def __init__(self, n_pages, page_size, max_seqs, max_pages):
        self.cfg = vfm_pages_config(int(n_pages), int(page_size), int(max_seqs), int(max_pages))
        self.page_size, self.max_pages = int(page_size), int(max_pages)
        n = C.c_size_t()
        _check(_lib_handle().vfm_pages_state_size(C.byref(self.cfg), C.byref(n)), "vfm_pages_state_size")
        self.state = np.zeros((n.value + 7) // 8, np.int64)      # 8-byte aligned
        _check(_lib_handle().vfm_pages_init(C.byref(self.cfg), self.state.ctypes.data, self.state.nbytes),
               "vfm_pages_init")

    def reserve(self, seq, n_tokens):
        _check(_lib_handle().vfm_pages_reserve(self.state.ctypes.data, int(seq), int(n_tokens)),
               "vfm_pages_reserve")

    def try_reserve(self, seq, n_tokens) -> bool:
        return _lib_handle().vfm_pages_reserve(self.state.ctypes.data, int(seq), int(n_tokens)) == VFM_OK

    def release(self, seq):
        _check(_lib_handle().vfm_pages_release(self.state.ctypes.data, int(seq)), "vfm_pages_release")

    def table(self, seqs, max_cols=None):
        seqs = np.ascontiguousarray(seqs, np.int32)
        cols = self.max_pages if max_cols is None else int(max_cols)
        out = np.empty((len(seqs), cols), np.int32)
        _check(_lib_handle().vfm_pages_table(self.state.ctypes.data, seqs.ctypes.data, len(seqs),
                                             out.ctypes.data, cols), "vfm_pages_table")
        return out

    def count(self, seq):
        h, f = C.c_int32(), C.c_int32()
        _check(_lib_handle().vfm_pages_count(self.state.ctypes.data, int(seq), C.byref(h), C.byref(f)),
               "vfm_pages_count")
        return h.value, f.value


# ---- batch-aware fair queueing (host scheduler, include/vfm_bfq.h) --------
class vfm_bfq_config(C.Structure):
    _fields_ = [("n_tasks", C.c_int32), ("b_max", C.c_int32), ("max_queued", C.c_int32),
                ("weight", C.POINTER(C.c_double)), ("batch_time", C.POINTER(C.c_double))]


class BFQ:
    """The library's BFQ scheduler on a host state buffer (numpy-owned)."""

    def __init__(self, weights, batch_time, b_max, max_queued=4096):
        self._w = np.ascontiguousarray(weights, np.float64)
        self._t = np.ascontiguousarray(batch_time, np.float64)
        self.b_max = int(b_max)
        self.cfg = vfm_bfq_config(len(self._w), self.b_max, int(max_queued),
                                  self._w.ctypes.data_as(C.POINTER(C.c_double)),
                                  self._t.ctypes.data_as(C.POINTER(C.c_double)))
        n = C.c_size_t()
        _check(_lib_handle().vfm_bfq_state_size(C.byref(self.cfg), C.byref(n)), "vfm_bfq_state_size")
        self.state = np.zeros((n.value + 7) // 8, np.float64)   # 8-byte aligned
        _check(_lib_handle().vfm_bfq_init(C.byref(self.cfg), self.state.ctypes.data, self.state.nbytes),
               "vfm_bfq_init")
        self._req = np.zeros(self.b_max, np.int64)
        self._task = np.zeros(self.b_max, np.int32)

    def enqueue(self, task, req, arrival, deadline=float("inf")):
        _check(_lib_handle().vfm_bfq_enqueue(self.state.ctypes.data, int(task), int(req), float(arrival),
                                             float(deadline)), "vfm_bfq_enqueue")

    def next_batch(self, now):
        """[(request id, task id)] of the next batch, in admission order."""
        n = C.c_int32()
        _check(_lib_handle().vfm_bfq_next_batch(self.state.ctypes.data, float(now), self._req.ctypes.data,
                                                self._task.ctypes.data, self.b_max, C.byref(n)),
               "vfm_bfq_next_batch")
        return [(int(self._req[k]), int(self._task[k])) for k in range(n.value)]

    def charge(self, task, service):
        _check(_lib_handle().vfm_bfq_charge(self.state.ctypes.data, int(task), float(service)),
               "vfm_bfq_charge")

    def queued(self, task):
        n = C.c_int32()
        _check(_lib_handle().vfm_bfq_queued(self.state.ctypes.data, int(task), C.byref(n)), "vfm_bfq_queued")
        return n.value

    def tags(self, task, k):
        s, f = C.c_double(), C.c_double()
        _check(_lib_handle().vfm_bfq_tags(self.state.ctypes.data, int(task), int(k), C.byref(s), C.byref(f)),
               "vfm_bfq_tags")
        return s.value, f.value
