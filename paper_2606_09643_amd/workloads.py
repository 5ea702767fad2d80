"""Seeded synthetic workloads for the mixed-task batched forward.

The five workloads below stand in for the paper's serving experiments
(representation FMs such as a ViT-B-sized vision encoder and a T5-large-sized
time-series encoder, and a 7B Llama-shaped token FM; Section 7.1, Table 2).
The paper's datasets, trained backbones and request traces are not available,
so every tensor here is drawn from a seeded generator with the shapes and
value distributions the workload names.

This module only *draws* numbers: task ids, lengths, weights, adapters, heads,
inputs and KV-cache contents.  It holds none of the forward arithmetic; both
the HIP path and the CPU oracle receive what it draws.

Seeding: ``numpy.random.SeedSequence([seed, workload.index])`` spawns one child
per stream in a fixed order (tasks, lengths, heads, backbone, adapters,
head weights, inputs, kv).  Per-layer streams are spawned from the backbone /
adapter / kv children, so any single layer can be regenerated on its own.
Tensors are drawn with a ``torch.Generator`` on the device they are requested
on, in float32, and then rounded to the workload dtype; the CPU and GPU
generators give different streams, so tests always hand the *same* drawn
tensors to both sides.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass

import numpy as np
import torch

DEFAULT_SEED = 20260601

# Projection order used throughout (matches the C ABI's projection enum).
PROJ = ("q", "k", "v", "o", "gate", "up", "down")
PROJ_INDEX = {p: i for i, p in enumerate(PROJ)}


@dataclass(frozen=True)
class Workload:
    index: int
    name: str
    dtype: str            # "f32" | "bf16": GEMM operand / activation type
    family: str           # "encoder" (pre-LN, GELU, biases) | "decoder" (RMSNorm, SwiGLU, RoPE)
    n_layers: int
    d: int
    n_heads: int
    head_dim: int
    d_ff: int
    n_tasks: int
    n_req: int
    rank: int
    lora_targets: tuple
    lora_scale: float
    zipf_s: float | None  # None: task ids uniform over the tasks
    seq_len: tuple        # (lo, hi), inclusive; tokens per request
    mode: str             # "prefill" | "decode"
    ctx: tuple | None     # decode: cached context length range (lo, hi), inclusive
    inputs: str           # "dense" | "patch" | "tokens"
    pool: str             # "mean" | "first" | "last" | "none"
    head: str             # "fixed:N" | "uniform:LO:HI" | "ts" | "none"
    vocab: int = 0
    patch: int = 0
    series_len: int = 0

    @property
    def causal(self) -> bool:
        return self.family == "decoder"

    @property
    def has_bias(self) -> bool:
        return self.family == "encoder"

    @property
    def norm(self) -> str:
        return "layer" if self.family == "encoder" else "rms"

    @property
    def norm_eps(self) -> float:
        return 1e-5 if self.family == "encoder" else 1e-6

    @property
    def rope_theta(self) -> float:
        return 10000.0 if self.family == "decoder" else 0.0

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    1: Workload(1, "tiny-encoder-f32", "f32", "encoder", 1, 256, 4, 64, 1024,
                n_tasks=4, n_req=16, rank=8, lora_targets=("q", "v"), lora_scale=2.0,
                zipf_s=None, seq_len=(64, 64), mode="prefill", ctx=None,
                inputs="dense", pool="mean", head="fixed:10"),
    2: Workload(2, "vitb-encoder-bf16", "bf16", "encoder", 12, 768, 12, 64, 3072,
                n_tasks=16, n_req=64, rank=16, lora_targets=("q", "k", "v", "o"),
                lora_scale=2.0, zipf_s=1.1, seq_len=(197, 197), mode="prefill",
                ctx=None, inputs="dense", pool="first", head="uniform:10:1000"),
    3: Workload(3, "t5l-timeseries-bf16", "bf16", "encoder", 24, 1024, 16, 64, 2816,
                n_tasks=32, n_req=128, rank=8, lora_targets=("q", "v"), lora_scale=2.0,
                zipf_s=1.2, seq_len=(64, 64), mode="prefill", ctx=None,
                inputs="patch", pool="mean", head="ts", patch=8, series_len=512),
    4: Workload(4, "llama7b-prefill-bf16", "bf16", "decoder", 32, 4096, 32, 128, 11008,
                n_tasks=64, n_req=32, rank=16, lora_targets=PROJ, lora_scale=2.0,
                zipf_s=1.1, seq_len=(128, 1024), mode="prefill", ctx=None,
                inputs="tokens", pool="none", head="none", vocab=32000),
    5: Workload(5, "llama7b-decode-bf16", "bf16", "decoder", 32, 4096, 32, 128, 11008,
                n_tasks=128, n_req=256, rank=16, lora_targets=PROJ, lora_scale=2.0,
                zipf_s=1.0, seq_len=(1, 1), mode="decode", ctx=(256, 2048),
                inputs="tokens", pool="last", head="fixed:8", vocab=32000),
}


def proj_dims(w: Workload, p: str) -> tuple:
    """(d_in, d_out) of projection ``p``."""
    if p in ("q", "k", "v", "o"):
        return w.d, w.d
    if p in ("gate", "up"):
        return w.d, w.d_ff
    if p == "down":
        return w.d_ff, w.d
    raise KeyError(p)


# --------------------------------------------------------------------------
# seed streams
# --------------------------------------------------------------------------
_STREAMS = ("tasks", "lengths", "heads", "backbone", "adapters", "head_w", "inputs", "kv")


def _children(w: Workload, seed: int) -> dict:
    kids = np.random.SeedSequence([seed, w.index]).spawn(len(_STREAMS))
    return dict(zip(_STREAMS, kids))


def _torch_gen(ss: np.random.SeedSequence, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(ss.generate_state(1, dtype=np.uint64)[0] & ((1 << 63) - 1)))
    return g


def _normal(shape, std, gen, device, dtype, mean=0.0):
    t = torch.empty(shape, dtype=torch.float32, device=device)
    t.normal_(mean=mean, std=std, generator=gen)
    return t.to(dtype)


def _layer_child(parent: np.random.SeedSequence, layer: int) -> np.random.SeedSequence:
    return np.random.SeedSequence(entropy=parent.entropy,
                                  spawn_key=tuple(parent.spawn_key) + (1000 + layer,))


# --------------------------------------------------------------------------
# batch composition
# --------------------------------------------------------------------------
def zipf_probs(n: int, s: float) -> np.ndarray:
    """Finite Zipf law over ranks 1..n: P(k) proportional to k**-s."""
    k = np.arange(1, n + 1, dtype=np.float64)
    p = k ** (-s)
    return p / p.sum()


@dataclass
class Batch:
    task_id: np.ndarray   # [n_req] int32, original request order
    seq_len: np.ndarray   # [n_req] int32
    ctx: np.ndarray | None  # [n_req] int32 (decode), cached tokens before the new one

    @property
    def n_req(self) -> int:
        return int(self.task_id.shape[0])

    @property
    def total_rows(self) -> int:
        return int(self.seq_len.sum())


def draw_batch(w: Workload, seed: int = DEFAULT_SEED) -> Batch:
    c = _children(w, seed)
    rt = np.random.default_rng(c["tasks"])
    if w.zipf_s is None:
        task = rt.integers(0, w.n_tasks, size=w.n_req)
    else:
        task = rt.choice(w.n_tasks, size=w.n_req, p=zipf_probs(w.n_tasks, w.zipf_s))
    rl = np.random.default_rng(c["lengths"])
    lo, hi = w.seq_len
    lens = rl.integers(lo, hi + 1, size=w.n_req)
    ctx = None
    if w.mode == "decode":
        clo, chi = w.ctx
        ctx = rl.integers(clo, chi + 1, size=w.n_req).astype(np.int32)
    return Batch(task.astype(np.int32), lens.astype(np.int32), ctx)


def draw_head_sizes(w: Workload, seed: int = DEFAULT_SEED) -> np.ndarray:
    """Output width of each task's linear head ([n_tasks] int32; 0 when no heads)."""
    c = _children(w, seed)
    r = np.random.default_rng(c["heads"])
    kind = w.head.split(":")
    if kind[0] == "none":
        return np.zeros(w.n_tasks, np.int32)
    if kind[0] == "fixed":
        return np.full(w.n_tasks, int(kind[1]), np.int32)
    if kind[0] == "uniform":
        return r.integers(int(kind[1]), int(kind[2]) + 1, size=w.n_tasks).astype(np.int32)
    if kind[0] == "ts":
        # half the tasks forecast 64 steps, the rest classify into 2..20 classes
        forecast = r.random(w.n_tasks) < 0.5
        cls = r.integers(2, 21, size=w.n_tasks)
        return np.where(forecast, 64, cls).astype(np.int32)
    raise ValueError(w.head)


def task_ranks(w: Workload) -> np.ndarray:
    return np.full(w.n_tasks, w.rank, np.int32)


# --------------------------------------------------------------------------
# backbone
# --------------------------------------------------------------------------
def backbone_layer(w: Workload, layer: int, device="cpu", seed: int = DEFAULT_SEED) -> dict:
    """One layer's shared weights, nn.Linear layout ``[d_out, d_in]``.

    Linear weights ~ N(0, 1/sqrt(d_model)) (std); encoder biases ~ N(0, 0.02);
    norm gains 1 + 0.1 N(0,1), LayerNorm shifts 0.1 N(0,1).  Q, K and V are
    stored stacked as one ``[3d, d]`` matrix (rows q, then k, then v).
    """
    c = _children(w, seed)
    g = _torch_gen(_layer_child(c["backbone"], layer), device)
    dt = w.torch_dtype
    d, f = w.d, w.d_ff
    std = 1.0 / np.sqrt(d)
    out = {}
    out["norm1_w"] = _normal((d,), 0.1, g, device, dt, mean=1.0)
    out["norm1_b"] = _normal((d,), 0.1, g, device, dt) if w.norm == "layer" else None
    out["w_qkv"] = _normal((3 * d, d), std, g, device, dt)
    out["b_qkv"] = _normal((3 * d,), 0.02, g, device, dt) if w.has_bias else None
    out["w_o"] = _normal((d, d), std, g, device, dt)
    out["b_o"] = _normal((d,), 0.02, g, device, dt) if w.has_bias else None
    out["norm2_w"] = _normal((d,), 0.1, g, device, dt, mean=1.0)
    out["norm2_b"] = _normal((d,), 0.1, g, device, dt) if w.norm == "layer" else None
    out["w_gate"] = _normal((f, d), std, g, device, dt) if w.family == "decoder" else None
    out["w_up"] = _normal((f, d), std, g, device, dt)
    out["b_up"] = _normal((f,), 0.02, g, device, dt) if w.has_bias else None
    out["w_down"] = _normal((d, f), std, g, device, dt)
    out["b_down"] = _normal((d,), 0.02, g, device, dt) if w.has_bias else None
    return out


def final_norm(w: Workload, device="cpu", seed: int = DEFAULT_SEED) -> dict:
    c = _children(w, seed)
    g = _torch_gen(_layer_child(c["backbone"], 999), device)
    dt = w.torch_dtype
    return {"w": _normal((w.d,), 0.1, g, device, dt, mean=1.0),
            "b": _normal((w.d,), 0.1, g, device, dt) if w.norm == "layer" else None}


# --------------------------------------------------------------------------
# per-task adapters and heads
# --------------------------------------------------------------------------
@dataclass
class LayerAdapters:
    """LoRA factors of one layer for every task.

    ``A[p]`` is ``[n_tasks, max_rank, d_in]``; task t's factor is the leading
    ``rank[t]`` rows of ``A[p][t]``.  ``B[p]`` is ``[n_tasks, d_out * max_rank]``;
    task t's ``[d_out, rank[t]]`` factor is the leading ``d_out * rank[t]``
    entries of ``B[p][t]``, row-major.
    """
    rank: np.ndarray        # [n_tasks] int32 (host)
    scale: np.ndarray       # [n_tasks] float32 (host)
    A: dict                 # proj -> tensor
    B: dict                 # proj -> tensor
    max_rank: int

    def a(self, p: str, t: int) -> torch.Tensor:
        r = int(self.rank[t])
        return self.A[p][t, :r, :]

    def b(self, p: str, t: int) -> torch.Tensor:
        r = int(self.rank[t])
        d_out = self.B[p].shape[1] // max(self.max_rank, 1)
        return self.B[p][t, : d_out * r].view(d_out, r)


def adapters_layer(w: Workload, layer: int, device="cpu", seed: int = DEFAULT_SEED,
                   ranks: np.ndarray | None = None, b_std: float = 0.01,
                   targets: tuple | None = None) -> LayerAdapters:
    """LoRA A ~ N(0, 1/sqrt(d_model)), B ~ N(0, b_std); scale per task."""
    c = _children(w, seed)
    g = _torch_gen(_layer_child(c["adapters"], layer), device)
    ranks = task_ranks(w) if ranks is None else np.asarray(ranks, np.int32)
    rmax = int(ranks.max()) if ranks.size else 0
    targets = w.lora_targets if targets is None else targets
    dt = w.torch_dtype
    A, B = {}, {}
    for p in targets:
        d_in, d_out = proj_dims(w, p)
        A[p] = _normal((w.n_tasks, rmax, d_in), 1.0 / np.sqrt(w.d), g, device, dt)
        B[p] = _normal((w.n_tasks, d_out * rmax), b_std, g, device, dt)
    scale = np.full(w.n_tasks, w.lora_scale, np.float32)
    return LayerAdapters(ranks, scale, A, B, rmax)


@dataclass
class Heads:
    n_out: np.ndarray    # [n_tasks] int32
    W: list              # per task [n_out_t, d] (workload dtype) or None
    b: list              # per task [n_out_t] (workload dtype) or None


def heads(w: Workload, device="cpu", seed: int = DEFAULT_SEED) -> Heads:
    """Per-task linear heads: W ~ N(0, 1/sqrt(d)), b ~ N(0, 0.02)."""
    n_out = draw_head_sizes(w, seed)
    c = _children(w, seed)
    g = _torch_gen(c["head_w"], device)
    dt = w.torch_dtype
    Ws, bs = [], []
    for t in range(w.n_tasks):
        n = int(n_out[t])
        if n == 0:
            Ws.append(None)
            bs.append(None)
            continue
        Ws.append(_normal((n, w.d), 1.0 / np.sqrt(w.d), g, device, dt))
        bs.append(_normal((n,), 0.02, g, device, dt))
    return Heads(n_out, Ws, bs)


# --------------------------------------------------------------------------
# inputs
# --------------------------------------------------------------------------
def dense_inputs(w: Workload, batch: Batch, device="cpu", seed: int = DEFAULT_SEED) -> torch.Tensor:
    """Token rows ~ N(0,1), ``[T, d]`` in original request order (workload dtype)."""
    c = _children(w, seed)
    g = _torch_gen(c["inputs"], device)
    return _normal((batch.total_rows, w.d), 1.0, g, device, w.torch_dtype)


def token_inputs(w: Workload, batch: Batch, device="cpu", seed: int = DEFAULT_SEED):
    """Token ids uniform over the vocabulary (``[T]`` int32, original order) and
    an embedding table ``[vocab, d]`` ~ N(0, 1)."""
    c = _children(w, seed)
    kid_ids, kid_emb = c["inputs"].spawn(2)
    ids = np.random.default_rng(kid_ids).integers(0, w.vocab, size=batch.total_rows)
    g = _torch_gen(kid_emb, device)
    emb = _normal((w.vocab, w.d), 1.0, g, device, w.torch_dtype)
    return torch.from_numpy(ids.astype(np.int32)).to(device), emb


def series_inputs(w: Workload, batch: Batch, device="cpu", seed: int = DEFAULT_SEED):
    """Time-series inputs: random walk (step std 0.05) plus a sinusoid of
    amplitude U(0.5, 2), period U(8, 128) and phase U(0, 2 pi), plus white
    noise of std 0.1; ``series_len`` samples per request, cut into
    ``series_len / patch`` patches.  Returns the patches ``[T, patch]`` float32
    (original order), the patch-embedding weight ``[d, patch]`` ~ N(0, 1/sqrt(patch))
    and bias ``[d]`` ~ N(0, 0.02) (workload dtype)."""
    c = _children(w, seed)
    kid_s, kid_w = c["inputs"].spawn(2)
    r = np.random.default_rng(kid_s)
    n, L = batch.n_req, w.series_len
    t = np.arange(L, dtype=np.float64)
    walk = np.cumsum(r.normal(0.0, 0.05, size=(n, L)), axis=1)
    amp = r.uniform(0.5, 2.0, size=(n, 1))
    period = r.uniform(8.0, 128.0, size=(n, 1))
    phase = r.uniform(0.0, 2 * np.pi, size=(n, 1))
    noise = r.normal(0.0, 0.1, size=(n, L))
    series = walk + amp * np.sin(2 * np.pi * t / period + phase) + noise
    patches = series.reshape(n * (L // w.patch), w.patch).astype(np.float32)
    g = _torch_gen(kid_w, device)
    W = _normal((w.d, w.patch), 1.0 / np.sqrt(w.patch), g, device, w.torch_dtype)
    b = _normal((w.d,), 0.02, g, device, w.torch_dtype)
    return torch.from_numpy(patches).to(device), W, b


def multichannel_series_inputs(w: Workload, batch: Batch, n_channels: int, patch: int, device="cpu",
                               seed: int = DEFAULT_SEED):
    """Multi-channel time series (e.g. the 3-channel physiological signals of
    the paper's MOMENT pipeline example): every channel of every request drawn
    with the recipe of ``series_inputs`` (random walk + sinusoid + noise),
    ``seq_len * patch`` samples per channel.  Returns the series float32 flat,
    requests in original order, each ``[n_channels, seq_len * patch]``
    channel-major, and a patch-embedding weight ``[d, patch]`` ~ N(0, 1/sqrt(patch))
    with bias ``[d]`` ~ N(0, 0.02) (workload dtype)."""
    c = _children(w, seed)
    kid_s, kid_w = np.random.SeedSequence(c["inputs"].generate_state(2)).spawn(2)
    r = np.random.default_rng(kid_s)
    parts = []
    for n_rows in batch.seq_len:
        L = int(n_rows) * patch
        t = np.arange(L, dtype=np.float64)
        walk = np.cumsum(r.normal(0.0, 0.05, size=(n_channels, L)), axis=1)
        amp = r.uniform(0.5, 2.0, size=(n_channels, 1))
        period = r.uniform(8.0, 128.0, size=(n_channels, 1))
        phase = r.uniform(0.0, 2 * np.pi, size=(n_channels, 1))
        noise = r.normal(0.0, 0.1, size=(n_channels, L))
        parts.append((walk + amp * np.sin(2 * np.pi * t / period + phase) + noise).ravel())
    series = np.concatenate(parts).astype(np.float32)
    g = _torch_gen(kid_w, device)
    W = _normal((w.d, patch), 1.0 / np.sqrt(patch), g, device, w.torch_dtype)
    b = _normal((w.d,), 0.02, g, device, w.torch_dtype)
    return torch.from_numpy(series).to(device), W, b


def kv_offsets(batch: Batch) -> np.ndarray:
    """Slot offset of each request's cache (original order); request i owns
    ``ctx[i] + 1`` slots, the last one for the token being decoded."""
    cap = batch.ctx.astype(np.int64) + 1
    off = np.zeros(batch.n_req, np.int64)
    off[1:] = np.cumsum(cap)[:-1]
    return off


def kv_cache_layer(w: Workload, batch: Batch, layer: int, device="cpu",
                   seed: int = DEFAULT_SEED):
    """Synthetic cached K and V (already rotated) ~ N(0,1), ``[sum(ctx+1), d]``
    each; the slot after each request's context is left zero."""
    c = _children(w, seed)
    g = _torch_gen(_layer_child(c["kv"], layer), device)
    total = int((batch.ctx.astype(np.int64) + 1).sum())
    k = _normal((total, w.d), 1.0, g, device, w.torch_dtype)
    v = _normal((total, w.d), 1.0, g, device, w.torch_dtype)
    off = kv_offsets(batch) + batch.ctx
    idx = torch.from_numpy(off).to(device)
    k[idx] = 0
    v[idx] = 0
    return k, v
