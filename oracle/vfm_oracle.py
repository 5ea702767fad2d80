"""Plain fp64 CPU oracle of FMplex's mixed-task batched forward.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
``bench.py``'s cpu_baseline leg may import this module.  The product path (the
HIP library and its binding) never imports, links or calls it, and this module
imports nothing from the product package.

What it computes (the paper, Section 2.3 "deployment sharing" and Section 4.2
"Batch-aware Fair Scheduling", last paragraph, with example (c) of Fig. 5):
requests of several tasks are batched through ONE shared backbone, and each
task's adapter difference is then applied to that task's requests only.  That
batching is a re-association of running every request through its own task's
customised model, i.e. the backbone with the task's LoRA adapter (Hu et al.,
cited in Section 2.2; PEFT's LoraConfig in Appendix A) followed by the task's
decoder head (Section 2.2).  So the oracle is that definition written out, one
request at a time, in float64:

    per layer:  h  = Norm1(x)
                y_P = h W_P^T + b_P + s_t (h A_{t,P}^T) B_{t,P}^T     (unmerged LoRA)
                attention over the request's own rows only
                x  = x + attn W_O^T + b_O (+ LoRA_O)
                h2 = Norm2(x)
                encoder:  u = GELU_erf(h2 W_up^T + b_up)
                decoder:  u = SiLU(h2 W_gate^T + d_gate) * (h2 W_up^T + d_up)
                x  = x + u W_down^T + b_down (+ LoRA_down)
    then final norm, pooling per request, and the task's linear head.

A task's pipeline may also carry an input-side encoder (a linear channel
combiner, C channels to one, ahead of the shared patch embedding) and an MLP
decoder head in place of the linear one (Section 4.3's pipeline example).

The backbone architectures (pre-LN ViT/T5-style encoder; Llama-style decoder
with RMSNorm, RoPE and SwiGLU) are the standard ones of the backbones the paper
serves (Table 2); the paper defines none of their arithmetic itself.  Where the
paper is silent this module takes these readings: LayerNorm eps 1e-5 with the
biased variance, RMSNorm eps 1e-6, exact-erf GELU, rotate-half RoPE with base
10000, decode attending to its ctx cached keys plus itself, and pooling per
workload (mean, first token or the decoded token).

Pins (tests/test_oracle_pins.py): plan vs brute force; merged == unmerged LoRA;
zero rank / zero B == bare backbone; LoRA closed form on unit vectors; encoder
layer vs torch's TransformerEncoderLayer; decoder layer vs transformers'
LlamaDecoderLayer; RoPE vs the complex-rotation form; attention special cases;
decode step == last prefill row; batched re-association == per-request
definition; MLP head and channel combiner on hand-worked examples and their
reductions to the linear head / a single channel.  Every function here is
pinned by at least one of them.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf

F64 = np.float64


# --------------------------------------------------------------------------
# a0: the plan (integer, bit-exact)
# --------------------------------------------------------------------------
def plan(task_id, seq_len, n_tasks, ctx=None, n_out=None) -> dict:
    """Segment a batch by task (Section 4.2: the scheduler's batch holds
    requests of several vFMs; the adapter difference is applied per task).

    Requests are ordered by task id ascending, ties kept in arrival order
    (a stable counting sort).  Returns int64 arrays:
      order[p]      original index of the request at plan position p
      task[p]       its task
      cu_seqlens    row offsets in plan order (n_req + 1)
      seg_req[t]    first plan position of task t (n_tasks + 1)
      seg_row[t]    first row of task t (n_tasks + 1)
      cu_orig       row offsets in original order (n_req + 1)
      pos[row]      position of each plan-order row within its request
                    (decode: offset by the cached context length)
      row_req[row]  plan position owning each row
      logit_off     output offsets in ORIGINAL order (n_req + 1): exclusive
                    scan of the head width of each request's task
    """
    task_id = [int(t) for t in task_id]
    seq_len = [int(n) for n in seq_len]
    n_req = len(task_id)
    for t in task_id:
        if not 0 <= t < n_tasks:
            raise ValueError("task id out of range")
    counts = [0] * n_tasks
    for t in task_id:
        counts[t] += 1
    seg_req = [0] * (n_tasks + 1)
    for t in range(n_tasks):
        seg_req[t + 1] = seg_req[t] + counts[t]
    nxt = list(seg_req[:n_tasks])
    order = [0] * n_req
    for i, t in enumerate(task_id):
        order[nxt[t]] = i
        nxt[t] += 1
    cu = [0] * (n_req + 1)
    for p in range(n_req):
        cu[p + 1] = cu[p] + seq_len[order[p]]
    seg_row = [cu[seg_req[t]] for t in range(n_tasks + 1)]
    cu_orig = [0] * (n_req + 1)
    for i in range(n_req):
        cu_orig[i + 1] = cu_orig[i] + seq_len[i]
    pos, row_req = [], []
    for p in range(n_req):
        base = int(ctx[order[p]]) if ctx is not None else 0
        for j in range(seq_len[order[p]]):
            pos.append(base + j)
            row_req.append(p)
    logit_off = [0] * (n_req + 1)
    for i in range(n_req):
        w = int(n_out[task_id[i]]) if n_out is not None else 0
        logit_off[i + 1] = logit_off[i] + w
    a = lambda v: np.asarray(v, dtype=np.int64)
    return {"order": a(order), "task": a([task_id[i] for i in order]),
            "cu_seqlens": a(cu), "seg_req": a(seg_req), "seg_row": a(seg_row),
            "cu_orig": a(cu_orig), "pos": a(pos), "row_req": a(row_req),
            "logit_off": a(logit_off)}


# --------------------------------------------------------------------------
# elementary operations of the backbone
# --------------------------------------------------------------------------
def layer_norm(x, g, b, eps):
    """LayerNorm over the last axis with the biased variance."""
    x = np.asarray(x, F64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    y = (x - mu) / np.sqrt(var + eps) * g
    return y + b if b is not None else y


def rms_norm(x, g, eps):
    """RMSNorm: x / sqrt(mean(x^2) + eps) * g."""
    x = np.asarray(x, F64)
    return x / np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps) * g


def norm(x, g, b, kind, eps):
    return layer_norm(x, g, b, eps) if kind == "layer" else rms_norm(x, g, eps)


def linear(x, W, b=None):
    """nn.Linear convention: W is [d_out, d_in]; y = x W^T + b."""
    y = np.asarray(x, F64) @ np.asarray(W, F64).T
    return y + b if b is not None else y


def lora_delta(x, A, B, scale):
    """LoRA difference of one task on one projection (Hu et al.; Section 2.2):
    scale * (x A^T) B^T with A [r, d_in], B [d_out, r].  Rank 0 gives zeros."""
    x = np.asarray(x, F64)
    if A is None or A.shape[0] == 0:
        return np.zeros((x.shape[0], B.shape[0] if B is not None else 0), F64)
    return scale * ((x @ np.asarray(A, F64).T) @ np.asarray(B, F64).T)


def gelu(x):
    """Exact (erf) GELU."""
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def silu(x):
    return x / (1.0 + np.exp(-x))


def rope(x, pos, n_heads, head_dim, theta):
    """Rotary embedding, rotate-half convention: within each head the pair
    (i, i + head_dim/2) is rotated by pos * theta**(-2i/head_dim)."""
    x = np.asarray(x, F64).reshape(x.shape[0], n_heads, head_dim)
    half = head_dim // 2
    inv = theta ** (-2.0 * np.arange(half, dtype=F64) / head_dim)
    ang = np.asarray(pos, F64)[:, None] * inv[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    a, b = x[..., :half], x[..., half:]
    out = np.concatenate([a * c - b * s, a * s + b * c], axis=-1)
    return out.reshape(x.shape[0], n_heads * head_dim)


def softmax_rows(s):
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=-1, keepdims=True)


def attention(q, k, v, n_heads, head_dim, causal=False, q_offset=0):
    """Scaled dot-product attention of one request, per head.

    q [Lq, d], k/v [Lk, d].  Causal: query row i (absolute position
    q_offset + i) sees keys 0..q_offset + i.
    """
    q = np.asarray(q, F64)
    k = np.asarray(k, F64)
    v = np.asarray(v, F64)
    Lq, Lk = q.shape[0], k.shape[0]
    out = np.empty((Lq, n_heads * head_dim), F64)
    for hh in range(n_heads):
        sl = slice(hh * head_dim, (hh + 1) * head_dim)
        s = q[:, sl] @ k[:, sl].T / math.sqrt(head_dim)
        if causal:
            qi = q_offset + np.arange(Lq)[:, None]
            kj = np.arange(Lk)[None, :]
            s = np.where(kj > qi, -np.inf, s)
        out[:, sl] = softmax_rows(s) @ v[:, sl]
    return out


# --------------------------------------------------------------------------
# one backbone layer, one request (the definition)
# --------------------------------------------------------------------------
def _split_qkv(W):
    d = W["w_qkv"].shape[1]
    w = np.asarray(W["w_qkv"], F64)
    b = W.get("b_qkv")
    bq = bk = bv = None
    if b is not None:
        b = np.asarray(b, F64)
        bq, bk, bv = b[:d], b[d:2 * d], b[2 * d:]
    return (w[:d], bq), (w[d:2 * d], bk), (w[2 * d:], bv)


def _proj(x, W, b, adapter, name):
    y = linear(x, W, b)
    if adapter is not None and name in adapter:
        A, B, s = adapter[name]
        y = y + lora_delta(x, A, B, s)
    return y


def layer(spec, W, adapter, x, pos=None, kv=None):
    """One layer of the shared backbone for ONE request with its task's adapter.

    spec: dict with family ("encoder" | "decoder"), n_heads, head_dim, norm
          ("layer" | "rms"), eps, rope_theta (0 = none).
    W:    the layer's shared weights (arrays; biases / LN shifts may be None).
    adapter: {proj: (A [r, d_in], B [d_out, r], scale)} of the request's task,
          or None for the bare backbone.
    x:    [L, d] the request's rows.
    pos:  [L] positions (RoPE).
    kv:   decode only: (K_ctx [ctx, d], V_ctx [ctx, d]) cached, already rotated.
    Returns (x_new [L, d], k_rows [L, d], v_rows [L, d]); k_rows are rotated.
    """
    x = np.asarray(x, F64)
    H, dh = spec["n_heads"], spec["head_dim"]
    kind, eps = spec["norm"], spec["eps"]
    h = norm(x, W["norm1_w"], W.get("norm1_b"), kind, eps)
    (wq, bq), (wk, bk), (wv, bv) = _split_qkv(W)
    q = _proj(h, wq, bq, adapter, "q")
    k = _proj(h, wk, bk, adapter, "k")
    v = _proj(h, wv, bv, adapter, "v")
    if spec.get("rope_theta", 0.0):
        q = rope(q, pos, H, dh, spec["rope_theta"])
        k = rope(k, pos, H, dh, spec["rope_theta"])
    causal = spec["family"] == "decoder"
    if kv is not None:
        kc, vc = np.asarray(kv[0], F64), np.asarray(kv[1], F64)
        kk, vv = np.concatenate([kc, k]), np.concatenate([vc, v])
        a = attention(q, kk, vv, H, dh, causal=True, q_offset=kc.shape[0])
    else:
        a = attention(q, k, v, H, dh, causal=causal)
    x = x + _proj(a, W["w_o"], W.get("b_o"), adapter, "o")
    h2 = norm(x, W["norm2_w"], W.get("norm2_b"), kind, eps)
    if spec["family"] == "encoder":
        u = gelu(_proj(h2, W["w_up"], W.get("b_up"), adapter, "up"))
    else:
        g = _proj(h2, W["w_gate"], None, adapter, "gate")
        u = silu(g) * _proj(h2, W["w_up"], None, adapter, "up")
    x = x + _proj(u, W["w_down"], W.get("b_down"), adapter, "down")
    return x, k, v


def pool(xn, mode):
    """Pool a request's final-normed rows to one vector."""
    if mode == "mean":
        return xn.mean(axis=0)
    if mode == "first":
        return xn[0]
    if mode == "last":
        return xn[-1]
    raise ValueError(mode)


def head(pooled, W, b):
    """Task-specific linear head on the pooled backbone output (Section 2.2)."""
    return linear(pooled[None, :], W, b)[0]


def head_mlp(pooled, W1, b1, W, b, act="gelu"):
    """Task-specific two-layer MLP decoder head (Section 4.3's pipeline
    example: an MLP decoder with a hidden width on the backbone output):
    act(pooled W1^T + b1) W^T + b, act the exact-erf GELU or ReLU."""
    h = linear(pooled[None, :], W1, b1)
    h = gelu(h) if act == "gelu" else np.maximum(h, 0.0)
    return linear(h, W, b)[0]


def channel_combine(x, W, b=None):
    """Task-specific input encoder: the linear channel combiner of Section
    4.3's pipeline example (C channels to one).  x [C, L] (a request's
    series, one row per channel), W [C], b scalar or None:
    s[l] = b + sum_c W[c] x[c, l]."""
    x = np.asarray(x, F64)
    s = np.asarray(W, F64) @ x
    return s + (float(np.asarray(b, F64).reshape(-1)[0]) if b is not None else 0.0)


def patch_embed(series, patch, W_pe, b_pe):
    """Shared patch embedding of a one-channel series: cut into consecutive
    patches of `patch` samples, each mapped to W_pe p + b_pe."""
    series = np.asarray(series, F64)
    return linear(series.reshape(-1, patch), W_pe, b_pe)


def final(spec, fn_w, fn_b, x):
    return norm(x, fn_w, fn_b, spec["norm"], spec["eps"])


# --------------------------------------------------------------------------
# the method's re-association (self-test of the oracle, not the definition)
# --------------------------------------------------------------------------
def merged_adapter_weights(W, A, B, scale):
    """W + scale * B A: the task's customised weight, for the merged self-test."""
    return np.asarray(W, F64) + scale * (np.asarray(B, F64) @ np.asarray(A, F64))


def batched_projection(x_rows, W, b, seg_row, adapters_by_task, name):
    """Shared projection for ALL rows at once, then each task's LoRA difference
    added on its own contiguous row segment (Section 4.2, adapter handling).
    x_rows are in plan order; seg_row[t]..seg_row[t+1] are task t's rows."""
    y = linear(x_rows, W, b)
    n_tasks = len(seg_row) - 1
    for t in range(n_tasks):
        r0, r1 = int(seg_row[t]), int(seg_row[t + 1])
        ad = adapters_by_task[t]
        if r1 > r0 and ad is not None and name in ad:
            A, B, s = ad[name]
            y[r0:r1] += lora_delta(x_rows[r0:r1], A, B, s)
    return y


def batched_layer(spec, W, adapters_by_task, x_rows, pl):
    """The whole batch through one layer the way the method runs it: norms and
    shared projections over all rows in plan order, LoRA per task segment,
    attention per request.  Prefill only."""
    H, dh = spec["n_heads"], spec["head_dim"]
    kind, eps = spec["norm"], spec["eps"]
    seg, cu = pl["seg_row"], pl["cu_seqlens"]
    x = np.asarray(x_rows, F64)
    h = norm(x, W["norm1_w"], W.get("norm1_b"), kind, eps)
    (wq, bq), (wk, bk), (wv, bv) = _split_qkv(W)
    q = batched_projection(h, wq, bq, seg, adapters_by_task, "q")
    k = batched_projection(h, wk, bk, seg, adapters_by_task, "k")
    v = batched_projection(h, wv, bv, seg, adapters_by_task, "v")
    if spec.get("rope_theta", 0.0):
        q = rope(q, pl["pos"], H, dh, spec["rope_theta"])
        k = rope(k, pl["pos"], H, dh, spec["rope_theta"])
    a = np.empty_like(q)
    for p in range(len(cu) - 1):
        sl = slice(int(cu[p]), int(cu[p + 1]))
        a[sl] = attention(q[sl], k[sl], v[sl], H, dh, causal=spec["family"] == "decoder")
    x = x + batched_projection(a, W["w_o"], W.get("b_o"), seg, adapters_by_task, "o")
    h2 = norm(x, W["norm2_w"], W.get("norm2_b"), kind, eps)
    if spec["family"] == "encoder":
        u = gelu(batched_projection(h2, W["w_up"], W.get("b_up"), seg, adapters_by_task, "up"))
    else:
        g = batched_projection(h2, W["w_gate"], None, seg, adapters_by_task, "gate")
        u = silu(g) * batched_projection(h2, W["w_up"], None, seg, adapters_by_task, "up")
    return x + batched_projection(u, W["w_down"], W.get("b_down"), seg, adapters_by_task, "down")


# --------------------------------------------------------------------------
# error measure used by every parity test
# --------------------------------------------------------------------------
def row_rel_error(got, ref):
    """Max over rows of max_j |got - ref| / max_j |ref| (row-normwise relative
    error).  Rows whose reference is all zero use an absolute measure."""
    got = np.asarray(got, F64).reshape(np.asarray(ref).shape[0], -1)
    ref = np.asarray(ref, F64).reshape(got.shape[0], -1)
    if ref.size == 0:
        return 0.0
    num = np.abs(got - ref).max(axis=1)
    den = np.abs(ref).max(axis=1)
    den = np.where(den > 0, den, 1.0)
    return float((num / den).max())
