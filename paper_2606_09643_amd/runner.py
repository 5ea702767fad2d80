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


def page_kv_cache(kv: KVCache, batch: wl.Batch, page_size, seed=0):
    """Moves every layer of a contiguous decode cache into a paged pool
    (pages in random order), freeing the contiguous copy layer by layer;
    returns the per-layer B.PagedKV."""
    n_tok = batch.ctx.astype(np.int64) + batch.seq_len
    out = []
    for li in range(len(kv.k)):
        kp, vp, table = paged_from_contiguous(kv.k[li], kv.v[li], kv.kv_start, n_tok, page_size,
                                              np.random.default_rng(seed + li))
        kv.k[li] = kv.v[li] = None
        torch.cuda.empty_cache()        # the next layer's pool reuses this layer's memory
        out.append(B.PagedKV(kp, vp, page_size, table))
    return out


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
        self.paged = None               # per layer B.PagedKV: the layers read a paged cache instead
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
        if self.paged is not None:
            B.vfm_layer_forward_paged(self.m.cfg, self.m.c_layers[li], self.m.lora_c(li), self.pb.c, self.x,
                                      self.paged[li], self.ws, stream)
            return
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


class _Seq:
    __slots__ = ("rid", "task", "prompt", "max_new", "slot", "cached", "generated", "budget", "row")

    def __init__(self, rid, task, prompt, max_new, page_size):
        self.rid, self.task = rid, int(task)
        self.prompt = np.asarray(prompt, np.int32)
        self.max_new = int(max_new)
        self.slot = -1
        self.cached = 0                 # tokens whose K / V are in the pages
        self.generated = []             # (step, index in that step's batch) of each new token
        self.row = -1                   # index in the latest step's batch
        # pages for every token that will ever be written (the last generated one never is)
        self.budget = -(-(len(self.prompt) + self.max_new - 1) // page_size)


class ContinuousBatcher:
    """Iteration-level (continuous) batching of a token-based FM over a paged
    KV cache.  Every step runs ONE mixed batch through all layers: the newly
    admitted prompts (ctx 0, their whole prompt) and one decode row for each
    running sequence (ctx = its cached tokens), then the final norm, each
    request's task head (pooled on its last row) and a greedy pick of its next
    token.  Pages come from the library's allocator as sequences grow and go
    back the moment a sequence finishes.

    Admission is FIFO, or BFQ order when a B.BFQ scheduler is given (its
    batches are taken whole and their requests join in that order as they
    fit, before any later batch is formed); with BFQ,
    every step also charges each task its decode rows times `token_time`
    (token-level work in service-time units), so tasks whose sequences keep
    generating fall back in the order of the prompts still waiting.  A prompt
    is admitted only when a sequence slot is free, its tokens fit the step's
    token budget, and the pages it will ever need fit next to those the
    running sequences may still need, so a running sequence never waits for
    a page (no preemption).  The host decides only the schedule; every row
    of the step is computed by the library's kernels."""

    def __init__(self, model: Model, emb, page_size=64, n_pages=1024, max_seqs=256, max_step_tokens=8192,
                 max_pages=None, bfq=None, token_time=1.0, chunk_prompts=None, record=False, device="cuda"):
        w = model.w
        self.m, self.emb, self.device = model, emb, device
        self.page_size, self.n_pages = int(page_size), int(n_pages)
        self.max_seqs, self.max_step_tokens = int(max_seqs), int(max_step_tokens)
        self.max_pages = int(max_pages) if max_pages is not None else self.n_pages
        self.alloc = B.PageAllocator(self.n_pages, self.page_size, self.max_seqs, self.max_pages)
        shape = (w.n_heads, self.n_pages * self.page_size, w.head_dim)
        self.k = [torch.zeros(shape, dtype=w.torch_dtype, device=device) for _ in range(model.n_layers)]
        self.v = [torch.zeros(shape, dtype=w.torch_dtype, device=device) for _ in range(model.n_layers)]
        self.cfg = B.vfm_cfg.from_buffer_copy(model.cfg)
        self.cfg.attn = B.VFM_ATTN_MIXED
        self.bfq, self.record, self.token_time = bfq, record, float(token_time)
        # prompt chunks after cached tokens run on the bf16 path only
        self.chunk = (w.dtype == "bf16") if chunk_prompts is None else bool(chunk_prompts)
        self.waiting, self.running, self.done = [], [], {}
        self.requests = {}
        self.free_slots = list(range(self.max_seqs - 1, -1, -1))
        self.committed = 0              # pages the running sequences hold or may still take
        self.ws = torch.empty(0, dtype=torch.uint8, device=device)
        self.steps = 0
        self.trace = []                 # per step: [(rid, logits)] when record is set
        self._picks, self._prev_nxt, self._keep = [], None, None
        self._ready = []                # taken from BFQ, not yet admitted (in its order)

    def submit(self, rid, task, prompt, max_new, now=0.0):
        s = _Seq(rid, task, prompt, max_new, self.page_size)
        if s.budget > self.max_pages or len(s.prompt) < 1 or s.max_new < 1:
            raise ValueError(f"request {rid}: needs {s.budget} pages (max {self.max_pages}) or is empty")
        self.requests[rid] = s
        if self.bfq is not None:
            self.bfq.enqueue(s.task, rid, now)
        self.waiting.append(s)

    def _fits(self, s, tokens):
        first = 1 if self.chunk else len(s.prompt)   # tokens it needs in this step
        return (self.free_slots and tokens + first <= self.max_step_tokens
                and self.committed + s.budget <= self.n_pages)

    def _admit_one(self, s):
        s.slot = self.free_slots.pop()
        self.committed += s.budget
        self.waiting.remove(s)
        self.running.append(s)

    def _admit(self, now):
        # rows already claimed this step: a decode row per decoding sequence and
        # the next chunk of every sequence still in its prompt
        tokens = 0
        for s in self.running:
            tokens += 1 if s.cached >= len(s.prompt) else min(len(s.prompt) - s.cached,
                                                              max(self.max_step_tokens - tokens, 0))
        new = []
        if self.bfq is None:
            for s in list(self.waiting):
                if not self._fits(s, tokens):
                    break
                self._admit_one(s)
                new.append(s)
                tokens += min(len(s.prompt), self.max_step_tokens - tokens)
            return new
        # BFQ: batches come whole in tag order; their requests join as
        # they fit (slot, token budget, pages), the rest first in later steps
        while True:
            if not self._ready:
                got = self.bfq.next_batch(now) if self.waiting else []
                if not got:
                    break
                self._ready = [self.requests[rid] for rid, _ in got]
            s = self._ready[0]
            if not self._fits(s, tokens):
                break
            self._ready.pop(0)
            self._admit_one(s)
            new.append(s)
            tokens += min(len(s.prompt), self.max_step_tokens - tokens)
        return new

    def _h2d(self, arr):
        """Host array -> device without waiting for the stream (pinned staging)."""
        return torch.from_numpy(np.ascontiguousarray(arr)).pin_memory().to(self.device, non_blocking=True)

    def step(self, now=0.0):
        """One continuous-batching step; returns the ids of the requests that finished.

        Nothing here waits for the GPU (unless `record` is set): a decode
        row's input token is gathered on the device from the previous step's
        greedy picks, the host copies go through pinned memory, and a
        sequence finishes by its token count, so the host plans step n + 1
        while the GPU still runs step n.  Token values are read back by
        `tokens()`."""
        new = self._admit(now)
        old = [s for s in self.running if s not in new]
        # decoding sequences first (their input is their last pick, on the
        # device), then the sequences still in their prompt, each with its
        # next chunk of the step's token budget (the whole rest of the prompt
        # when prompts are not chunked)
        dec = [s for s in old if s.cached >= len(s.prompt)]
        budget = self.max_step_tokens - len(dec)
        chunks = []
        for s in [s for s in old if s.cached < len(s.prompt)] + new:
            n = len(s.prompt) - s.cached
            if self.chunk:
                n = min(n, budget)
            if n <= 0:
                continue
            chunks.append((s, n))
            budget -= n
        batch = dec + [s for s, _ in chunks]
        if not batch:
            return []
        w = self.m.w
        task = np.array([s.task for s in batch], np.int32)
        lens = np.array([1] * len(dec) + [n for _, n in chunks], np.int32)
        ctx = np.array([s.cached for s in batch], np.int32)
        for s, c, n in zip(batch, ctx, lens):
            self.alloc.reserve(s.slot, int(c) + int(n))
        slots = np.array([s.slot for s in batch], np.int32)
        table = self.alloc.table(slots, max(int(self.alloc.count(int(x))[0]) for x in slots))
        table_dev = self._h2d(table)
        pb = B.Batch(task, lens, w.n_tasks, ctx_len=ctx, n_out=self.m.heads.n_out, device=self.device,
                     non_blocking=True)
        need = max(B.vfm_workspace_size(self.cfg, pb.c, self.m.lora_c(i)) for i in range(self.m.n_layers))
        if need > self.ws.numel():
            self.ws = torch.empty(need, dtype=torch.uint8, device=self.device)
        x = torch.empty(pb.T, w.d, dtype=torch.float32, device=self.device)
        # input tokens, original order: decode rows' last picks (on device), then the prompt chunks
        n_dec = len(dec)
        parts = []
        if n_dec:
            parts.append(self._prev_nxt[self._h2d(np.array([s.row for s in dec], np.int64))])
        if chunks:
            parts.append(self._h2d(np.concatenate([s.prompt[s.cached:s.cached + n] for s, n in chunks])
                                   .astype(np.int32)))
        ids_dev = torch.cat(parts) if len(parts) > 1 else parts[0]
        B.vfm_embed_forward(self.cfg, pb.c, B.VFM_EMBED_TOKENS, ids_dev, w.vocab, self.emb, None, x)
        tp = table.ctypes.data_as(B.C.POINTER(B.C.c_int32))     # one device table for every layer
        for li in range(self.m.n_layers):
            kv = B.vfm_kv_pages(self.k[li].data_ptr(), self.v[li].data_ptr(), self.n_pages, self.page_size,
                                table.shape[1], tp, table_dev.data_ptr())
            B.vfm_layer_forward_paged(self.cfg, self.m.c_layers[li], self.m.lora_c(li), pb.c, x, kv, self.ws)
        out = torch.empty(max(pb.total_outputs, 1), dtype=torch.float32, device=self.device)
        fn = self.m.final
        B.vfm_head_forward(self.cfg, fn["w"], fn.get("b"), self.m.head_tab.c, pb.c, x, out, self.ws)
        nxt = torch.empty(len(batch), dtype=torch.int32, device=self.device)
        B.vfm_greedy_tokens(pb.c, out, nxt)
        self._prev_nxt = nxt
        self._picks.append(nxt)
        self._keep = (pb, table, table_dev)            # host arrays the stream may still read
        if self.bfq is not None and n_dec:
            per_task = np.bincount(task[:n_dec], minlength=w.n_tasks)
            for t in np.nonzero(per_task)[0]:
                self.bfq.charge(int(t), float(per_task[t]) * self.token_time)
        o = out.cpu().numpy() if self.record else None
        off = pb.out_off() if self.record else None
        rec, finished = [], []
        for i, s in enumerate(batch):
            s.cached += int(lens[i])
            if s.cached < len(s.prompt):               # a chunk inside the prompt: no token yet
                continue
            s.generated.append((self.steps, i))
            s.row = i
            if self.record:
                rec.append((s.rid, o[off[i]:off[i + 1]].copy()))
            if len(s.generated) == s.max_new:
                self.alloc.release(s.slot)
                self.free_slots.append(s.slot)
                self.committed -= s.budget
                self.running.remove(s)
                self.done[s.rid] = s
                finished.append(s.rid)
        if self.record:
            self.trace.append(rec)
        self.steps += 1
        return finished

    def tokens(self):
        """{request id: generated token ids} of the finished requests (one read-back)."""
        if not self._picks:
            return {}
        flat = torch.cat(self._picks).cpu().numpy()
        base = np.concatenate([[0], np.cumsum([len(p) for p in self._picks])])
        return {rid: [int(flat[base[st] + i]) for st, i in s.generated] for rid, s in self.done.items()}

    def run(self, now=0.0):
        """Steps until every submitted request has finished."""
        while self.waiting or self.running:
            before = (len(self.waiting), len(self.running))
            self.step(now)
            if not self.running and (len(self.waiting), len(self.running)) == before:
                raise RuntimeError("a waiting request can never be admitted")
        return self.tokens()
