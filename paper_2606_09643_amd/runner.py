"""Drives the C ABI over a whole mixed-task forward: input rows -> every
backbone layer -> final norm, pooling and per-task heads.

Owns the device tensors (weights, per-task adapter and head tables, plan,
workspace) and issues the library calls in order on one stream; it performs
no arithmetic of its own.
"""
from __future__ import annotations

import numpy as np
import torch

from . import binding as B
from . import workloads as wl

_POOL = {"mean": B.VFM_POOL_MEAN, "first": B.VFM_POOL_FIRST, "last": B.VFM_POOL_LAST}


def cfg_for(w: wl.Workload) -> B.vfm_cfg:
    if w.mode == "decode":
        attn = B.VFM_ATTN_DECODE
    else:
        attn = B.VFM_ATTN_CAUSAL if w.causal else B.VFM_ATTN_BIDIR
    return B.make_cfg(B.VFM_BF16 if w.dtype == "bf16" else B.VFM_F32, w.d, w.n_heads, w.head_dim,
                      w.d_ff, B.VFM_NORM_LAYER if w.norm == "layer" else B.VFM_NORM_RMS,
                      B.VFM_MLP_GELU if w.family == "encoder" else B.VFM_MLP_SWIGLU, attn,
                      w.has_bias, w.norm_eps, w.rope_theta)


def lora_table(w: wl.Workload, ad: wl.LayerAdapters, device="cuda") -> B.LoraTable:
    factors = {p: ([ad.a(p, t) for t in range(w.n_tasks)], [ad.b(p, t) for t in range(w.n_tasks)])
               for p in ad.A}
    return B.LoraTable(w.n_tasks, ad.rank, ad.scale, factors, max_rank=ad.max_rank, device=device)


def head_table(w: wl.Workload, hd: wl.Heads, device="cuda") -> B.HeadTable:
    return B.HeadTable(hd.n_out, hd.W, hd.b, _POOL[w.pool], device=device)


class Model:
    """Backbone layers, per-task adapters and heads of a workload, on device."""

    def __init__(self, w: wl.Workload, device="cuda", seed=wl.DEFAULT_SEED, n_layers=None,
                 ranks=None, b_std=0.01, with_lora=True):
        self.w = w
        self.cfg = cfg_for(w)
        self.n_layers = w.n_layers if n_layers is None else n_layers
        self.layers = [wl.backbone_layer(w, i, device, seed) for i in range(self.n_layers)]
        self.c_layers = [B.layer_weights(W) for W in self.layers]
        self.adapters = [wl.adapters_layer(w, i, device, seed, ranks=ranks, b_std=b_std)
                         if with_lora else None for i in range(self.n_layers)]
        self.lora = [lora_table(w, a, device) if a is not None else None for a in self.adapters]
        self.final = wl.final_norm(w, device, seed)
        self.heads = wl.heads(w, device, seed) if w.head != "none" else None
        self.head_tab = head_table(w, self.heads, device) if self.heads is not None else None

    def lora_c(self, i):
        return self.lora[i].c if self.lora[i] is not None else None


class Inputs:
    """The workload's input tensors (original request order) and how to embed them."""

    def __init__(self, w: wl.Workload, batch: wl.Batch, device="cuda", seed=wl.DEFAULT_SEED):
        self.w = w
        if w.inputs == "dense":
            self.mode, self.src, self.width = B.VFM_EMBED_ROWS, wl.dense_inputs(w, batch, device, seed), w.d
            self.table = self.bias = None
        elif w.inputs == "tokens":
            ids, emb = wl.token_inputs(w, batch, device, seed)
            self.mode, self.src, self.width, self.table, self.bias = B.VFM_EMBED_TOKENS, ids, w.vocab, emb, None
        else:
            patches, W, b = wl.series_inputs(w, batch, device, seed)
            self.mode, self.src, self.width, self.table, self.bias = B.VFM_EMBED_PATCHES, patches, w.patch, W, b


class KVCache:
    """Per-layer cached K / V for the decode workload, in the library's
    head-major layout [n_heads, sum(ctx + 1), head_dim]."""

    def __init__(self, w: wl.Workload, batch: wl.Batch, n_layers, device="cuda", seed=wl.DEFAULT_SEED):
        self.kv_start = wl.kv_offsets(batch).astype(np.int32)
        self.slots = int((batch.ctx.astype(np.int64) + 1).sum())
        self.n_heads, self.head_dim = w.n_heads, w.head_dim
        self.k, self.v = [], []
        for i in range(n_layers):
            k, v = wl.kv_cache_layer(w, batch, i, device, seed)
            self.k.append(self._head_major(k))
            self.v.append(self._head_major(v))
            del k, v

    def _head_major(self, t):
        return t.view(t.shape[0], self.n_heads, self.head_dim).permute(1, 0, 2).contiguous()

    def rows(self, li, s0, n):
        """(K, V) of slots s0 .. s0 + n - 1 of layer li as [n, d] tensors."""
        def take(c):
            return c[:, s0:s0 + n, :].permute(1, 0, 2).reshape(n, self.n_heads * self.head_dim)
        return take(self.k[li]), take(self.v[li])


def paged_from_contiguous(kc, vc, kv_start, n_tok, page_size, rng, spare_pages=0):
    """A paged copy of a head-major cache: request i's slots kv_start[i] ..
    kv_start[i] + n_tok[i] - 1 go, in order, to ceil(n_tok[i] / page_size)
    pages drawn in random order from a pool with `spare_pages` unused ones.
    Returns (k_pool, v_pool, table [n_req, max_pages] int32)."""
    n_tok = np.asarray(n_tok, np.int64)
    need = (n_tok + page_size - 1) // page_size
    total = int(need.sum()) + int(spare_pages)
    perm = rng.permutation(total).astype(np.int32)
    table = np.zeros((len(n_tok), max(int(need.max()), 1)), np.int32)
    first = np.concatenate([[0], np.cumsum(need)[:-1]])
    for i in range(len(n_tok)):
        table[i, :need[i]] = perm[first[i]:first[i] + need[i]]
    req = np.repeat(np.arange(len(n_tok)), n_tok)
    pos = np.arange(int(n_tok.sum())) - np.repeat(np.cumsum(n_tok) - n_tok, n_tok)
    phys = table[req, pos // page_size].astype(np.int64) * page_size + pos % page_size
    src = np.asarray(kv_start, np.int64)[req] + pos
    H, _, hd = kc.shape
    dev = kc.device
    phys_t, src_t = torch.from_numpy(phys).to(dev), torch.from_numpy(src).to(dev)
    pools = []
    for c in (kc, vc):
        pool = torch.zeros(H, total * page_size, hd, dtype=c.dtype, device=dev)
        pool[:, phys_t] = c[:, src_t]
        pools.append(pool)
    return pools[0], pools[1], table


def make_batch(w: wl.Workload, batch: wl.Batch, heads: wl.Heads | None, kv: KVCache | None = None,
               device="cuda") -> B.Batch:
    return B.Batch(batch.task_id, batch.seq_len, w.n_tasks,
                   ctx_len=batch.ctx if w.mode == "decode" else None,
                   kv_start=kv.kv_start if kv is not None else None,
                   n_out=heads.n_out if heads is not None else None, device=device)


class Forward:
    """Preallocated buffers and the call sequence of one forward step."""

    def __init__(self, model: Model, pb: B.Batch, inputs: Inputs, kv: KVCache | None = None,
                 device="cuda"):
        self.m, self.pb, self.inp, self.kv = model, pb, inputs, kv
        w = model.w
        need = max(B.vfm_workspace_size(model.cfg, pb.c, model.lora_c(i)) for i in range(model.n_layers))
        self.ws = torch.empty(need, dtype=torch.uint8, device=device)
        self.x = torch.empty(pb.T, w.d, dtype=torch.float32, device=device)
        if model.head_tab is not None:
            self.out = torch.empty(max(pb.total_outputs, 1), dtype=torch.float32, device=device)
        else:
            self.out = torch.empty(pb.T, w.d, dtype=torch.float32, device=device)

    def embed(self, stream=None):
        i = self.inp
        B.vfm_embed_forward(self.m.cfg, self.pb.c, i.mode, i.src, i.width, i.table, i.bias, self.x, stream)

    def layer(self, li, stream=None):
        kc = self.kv.k[li] if self.kv is not None else None
        vc = self.kv.v[li] if self.kv is not None else None
        slots = self.kv.slots if self.kv is not None else 0
        B.vfm_layer_forward(self.m.cfg, self.m.c_layers[li], self.m.lora_c(li), self.pb.c, self.x,
                            kc, vc, slots, self.ws, stream)

    def head(self, stream=None):
        fn = self.m.final
        B.vfm_head_forward(self.m.cfg, fn["w"], fn["b"],
                           self.m.head_tab.c if self.m.head_tab is not None else None,
                           self.pb.c, self.x, self.out, self.ws, stream)

    def __call__(self, stream=None):
        self.embed(stream)
        for li in range(self.m.n_layers):
            self.layer(li, stream)
        self.head(stream)
        return self.out
