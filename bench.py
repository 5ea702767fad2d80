"""Benchmark of the mixed-task batched forward on one MI355X.

One step = one whole forward of a mixed batch: input rows -> every backbone
layer (shared projections + per-task LoRA + per-request attention) -> final
norm (and, where the workload has them, pooling and per-task heads).  Default
workload: the Llama-7B-shaped decoder prefill (32 layers, d 4096, SwiGLU
11008, RoPE, RMSNorm; 32 prompts of U[128, 1024] tokens over 64 tasks with
Zipf(1.1) task ids, LoRA rank 16 on all seven projections), the largest
configuration that fits one GPU, with every input resident in HBM.

Prints ONE JSON line.  `value` is tokens/s of the whole step from the median
of the timed steps (each step bracketed by its own pair of hipEvents on the
forward's stream); `roofline` is the dominant kernel's achieved rate
(algorithmic FLOPs or bytes per launch / its average duration from hipEvents
recorded around its launches inside the same timed region) against the
MI355X peak; `cpu_baseline` times the fp64 oracle on a bounded sample of the
same batch on this host's cores (all of them, then one).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3    # MI355X fp32 (matrix / vector)
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
METRIC = "mixed-task backbone forward tokens/s at 1 GPU; % of bf16 MFMA / HBM roofline"


# --------------------------------------------------------------------------
# algorithmic work (what the method must do; no padding or recomputation)
# --------------------------------------------------------------------------
def algorithmic_work(w, batch, ranks, heads_n_out):
    """Per-step FLOPs by kernel class and HBM bytes of the decode step."""
    T = batch.total_rows
    d, f, H, dh, L = w.d, w.d_ff, w.n_heads, w.head_dim, w.n_layers
    lens = batch.seq_len.astype(np.float64)
    rk = ranks[batch.task_id].astype(np.float64)          # rank of each request's task
    rows_r = float((lens * rk).sum())                      # sum over rows of their rank
    tgt = set(w.lora_targets)

    def lora(p, d_in, d_out):
        return 2.0 * rows_r * (d_in + d_out) if p in tgt else 0.0

    fl = {}
    fl["gemm_qkv"] = 2.0 * T * d * 3 * d + sum(2.0 * rows_r * d for p in ("q", "k", "v") if p in tgt)
    fl["gemm_o"] = 2.0 * T * d * d + (2.0 * rows_r * d if "o" in tgt else 0.0)
    n_up = 2 if w.family == "decoder" else 1
    fl["gemm_up"] = 2.0 * T * d * f * n_up + sum(2.0 * rows_r * f for p in ("gate", "up") if p in tgt)
    fl["gemm_down"] = 2.0 * T * f * d + (2.0 * rows_r * d if "down" in tgt else 0.0)
    fl["shrink"] = sum(2.0 * rows_r * (d if p != "down" else f) for p in tgt)
    if w.mode == "decode":
        keys = batch.ctx.astype(np.float64) + 1.0
        fl["attn"] = float((4.0 * keys * dh * H).sum())
    elif w.causal:
        fl["attn"] = float((2.0 * dh * H * lens * (lens + 1)).sum())
    else:
        fl["attn"] = float((4.0 * dh * H * lens * lens).sum())
    per_step = {k: v * L for k, v in fl.items()}
    head_flops = float(sum(2.0 * d * heads_n_out[t] for t in batch.task_id)) if heads_n_out is not None else 0.0
    total = sum(per_step.values()) + head_flops
    # decode bytes: KV read + write, weights once, adapters of distinct tasks, heads
    es = 2 if w.dtype == "bf16" else 4
    kv_read = float((batch.ctx.astype(np.float64) + 1).sum() * d * 2 * es) if w.mode == "decode" else 0.0
    weights = (3 * d * d + d * d + n_up * f * d + f * d) * es
    distinct = np.unique(batch.task_id)
    ad_bytes = 0.0
    for p in tgt:
        d_in, d_out = (d, d) if p in ("q", "k", "v", "o") else ((d, f) if p in ("gate", "up") else (f, d))
        ad_bytes += float(ranks[distinct].sum()) * (d_in + d_out) * es
    step_bytes = L * (kv_read + weights + ad_bytes)
    return {"per_launch_flops": fl, "step_flops": total, "kv_read_bytes_per_layer": kv_read,
            "step_bytes": step_bytes}


# --------------------------------------------------------------------------
# HBM traffic of the dominant kernel, from the committed counter summary
# --------------------------------------------------------------------------
def hbm_traffic(workload_name, cls):
    """Bytes per launch from rocprofv3 FETCH_SIZE / WRITE_SIZE passes, each
    scaled by the same counter's reading for a device copy of known size
    (profiles/hbm_traffic.json); None when there is no record for this
    kernel or its sources have changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    try:
        rec = json.load(open(path)).get(workload_name)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("class") != cls:
        return None
    h = hashlib.sha256()
    for src in rec["source"]:
        try:
            h.update(open(os.path.join(ROOT, src), "rb").read())
        except OSError:
            return None
    if h.hexdigest() != rec["source_sha256"]:
        return None
    return float(rec["traffic_bytes_per_launch"])


# --------------------------------------------------------------------------
# CPU baseline: the fp64 oracle on a bounded sample of the same batch
# --------------------------------------------------------------------------
def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def _baseline_sample(w, batch, pl):
    """Requests (original indices) the oracle is timed on, per workload: every
    request of the tiny encoder, 8 ViT-B requests, 16 time series, the
    shortest and the longest decoder prompt, 8 decode requests (the first
    ones in original order)."""
    n = batch.n_req
    if w.family == "decoder" and w.mode != "decode":
        lens = batch.seq_len
        return sorted({int(np.argmin(lens)), int(np.argmax(lens))})
    k = {"tiny-encoder-f32": n, "vitb-encoder-bf16": 8, "t5l-timeseries-bf16": 16}.get(w.name, 8)
    return list(range(min(k, n)))


def cpu_baseline(w, batch, model, inp, kv=None):
    """The fp64 oracle on whole requests of the same batch, layer by layer.

    The sample (_baseline_sample) runs every layer and the final norm / head
    on all of this host's cores (BLAS threads), then its first layer again
    on one core; each layer's weights (and, when decoding, the requests' KV
    slices) are converted to fp64 outside the timed regions.  Also reported:
    the whole batch's oracle time derived from the sample (scaled by tokens,
    marked derived) and the CPU model.
    """
    from oracle import vfm_oracle as O
    from tests.gpu_common import expected_embed, oracle_plan
    from tests.helpers import np64, oracle_adapter, oracle_weights, spec_of
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threadpool_limits = None
        cores = os.cpu_count()
    pl = oracle_plan(w, batch, model.heads.n_out if model.heads is not None else None)
    x_all = expected_embed(w, batch, inp, pl)
    spec = spec_of(w)
    cu = pl["cu_seqlens"]
    inv = np.argsort(pl["order"])
    sample = _baseline_sample(w, batch, pl)
    x0 = {i: x_all[int(cu[int(inv[i])]):int(cu[int(inv[i]) + 1])] for i in sample}
    del x_all
    xs = dict(x0)

    def kv_of(li, i):
        if kv is None:
            return None
        c, s0 = int(batch.ctx[i]), int(kv.kv_start[i])
        kr, vr = kv.rows(li, s0, c)
        return (np64(kr), np64(vr))

    def run_layer(Wn, li, i, x, kvp):
        p = int(inv[i])
        t = int(pl["task"][p])
        sl = slice(int(cu[p]), int(cu[p + 1]))
        return O.layer(spec, Wn, oracle_adapter(model.adapters[li], t), x, pos=pl["pos"][sl],
                       kv=kvp)[0]

    elapsed = 0.0
    W0 = None
    for li in range(w.n_layers):
        Wn = oracle_weights(model.layers[li])
        if li == 0:
            W0 = Wn
        kvs = {i: kv_of(li, i) for i in sample}
        t0 = time.perf_counter()
        for i in sample:
            xs[i] = run_layer(Wn, li, i, xs[i], kvs[i])
        elapsed += time.perf_counter() - t0
        del Wn
    fw, fb = np64(model.final["w"]), np64(model.final["b"])
    t0 = time.perf_counter()
    for i in sample:
        t = int(pl["task"][int(inv[i])])
        xn = O.final(spec, fw, fb, xs[i])
        if model.heads is not None:
            O.head(O.pool(xn, w.pool), np64(model.heads.W[t]), np64(model.heads.b[t]))
    elapsed += time.perf_counter() - t0
    tokens = int(sum(xs[i].shape[0] for i in sample))
    # one core: the sample's first layer, scaled to every layer (derived)
    single = None
    if threadpool_limits is not None:
        kvs = {i: kv_of(0, i) for i in sample}
        with threadpool_limits(limits=1):
            t0 = time.perf_counter()
            for i in sample:
                run_layer(W0, 0, i, x0[i], kvs[i])
            t1 = time.perf_counter() - t0
        single = {"value": tokens / (t1 * w.n_layers), "unit": "tokens/s", "cores": 1,
                  "layer_seconds": t1, "derived": f"layer 0 of the same sample timed on one core, "
                                                  f"scaled to {w.n_layers} layers"}
    total_tokens = int(batch.total_rows)
    return {"value": tokens / elapsed, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "cpu_model": _cpu_model(),
            "sample": f"requests {sample} of {batch.n_req} (original order), {tokens} tokens, "
                      f"all {w.n_layers} layers + final norm" + ("/head" if model.heads is not None else "")
                      + f", fp64 numpy, {elapsed:.1f} s",
            "seconds": elapsed,
            "single_core": single,
            "full_batch_seconds_derived": elapsed * total_tokens / tokens,
            "full_batch_note": f"derived: the sample's time scaled by tokens ({total_tokens} / {tokens})"}


def loop_bench(args):
    """Continuous batching of the 7B decoder workload's model (all layers,
    128 tasks with rank-16 LoRA on every projection, per-task heads): n
    requests with prompts of U[64, 512] tokens and U[32, 128] new tokens each,
    at most 256 running sequences, pages of 64 slots, prompts admitted FIFO
    (or by BFQ with --admission bfq) up to 8192 tokens per step.  Timed from the first step to the last request
    finishing, host scheduling and the per-step token read-back included."""
    import torch
    from paper_2606_09643_amd import binding as B
    from paper_2606_09643_amd import runner as R
    from paper_2606_09643_amd import workloads as wl
    w = wl.WORKLOADS[5]
    model = R.Model(w)
    one = wl.Batch(np.zeros(1, np.int32), np.ones(1, np.int32), None)
    _, emb = wl.token_inputs(w, one, "cuda")
    rng = np.random.default_rng(20260601)
    n = args.loop
    tasks = rng.choice(w.n_tasks, size=n, p=wl.zipf_probs(w.n_tasks, w.zipf_s))
    plen = rng.integers(64, 513, size=n)
    new = rng.integers(32, 129, size=n)
    page, max_seqs = 64, 256
    n_pages = max_seqs * ((512 + 128 + page - 1) // page)

    def make():
        bfq = None
        if args.admission == "bfq":
            # equal weights; T(b): a prompt step's time grows with its prompts (unit: one decode step)
            bfq = B.BFQ(np.ones(w.n_tasks), [0.0] + [1.0 + 0.25 * b for b in range(1, 17)], b_max=16)
        cb = R.ContinuousBatcher(model, emb, page_size=page, n_pages=n_pages, max_seqs=max_seqs,
                                 max_step_tokens=8192, max_pages=(512 + 128 + page - 1) // page, bfq=bfq,
                                 token_time=1.0 / max_seqs)
        for i in range(n):
            cb.submit(i, int(tasks[i]), rng.integers(0, w.vocab, size=int(plen[i])), int(new[i]))
        return cb
    warm = make()                                      # warm-up run (kernels, allocator caches)
    for _ in range(3):
        warm.step()
    del warm
    cb = make()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    cb.run()
    torch.cuda.synchronize()
    sec = time.perf_counter() - t0
    gen = int(new.sum())
    out = {"metric": "continuous-batching generated tokens/s at 1 GPU (paged KV, mixed prefill + decode steps)",
           "value": gen / sec, "unit": "tokens/s", "n_gpus": 1, "steps": cb.steps,
           "ms_per_step": sec * 1e3 / cb.steps, "higher_is_better": True, "vs_baseline": None,
           "dtype": "bf16", "data": "synthetic",
           "config": {"workload": w.name + " continuous batching", "requests": n,
                      "prompt_tokens": int(plen.sum()), "generated_tokens": gen, "max_running": max_seqs,
                      "page_size": page, "max_step_tokens": 8192, "admission": args.admission},
           "seconds": sec}
    print(json.dumps(out), flush=True)


def task_load_bench(args):
    """Time to load one task into a running ViT-B-shaped backbone: its LoRA
    factors for every layer (rank 16 on q/k/v/o) and its head (the table's widest),
    packed as one pinned host blob and copied in one transfer, then attached to
    the layers' adapter tables and the head table (vfm_lora_attach per layer,
    vfm_head_attach), on the forward's stream; timed from the first copy to
    the attached tables being visible to the next forward (stream
    synchronised), median of 50 loads."""
    import torch
    from paper_2606_09643_amd import binding as B
    from paper_2606_09643_amd import runner as R
    from paper_2606_09643_amd import workloads as wl
    w = wl.WORKLOADS[2]
    model = R.Model(w)
    r, t = w.rank, 1
    n_out = int(model.head_tab.c.max_out)        # the widest head of the table
    # the task's artifact as one pinned blob: every layer's A, B factors, then the head
    shapes = []
    for li in range(w.n_layers):
        for p in w.lora_targets:
            d_in, d_out = wl.proj_dims(w, p)
            shapes += [((li, p, "A"), (r, d_in)), ((li, p, "B"), (d_out, r))]
    shapes += [(("head", "W"), (n_out, w.d)), (("head", "b"), (n_out,))]
    sizes = [int(np.prod(sh)) for _, sh in shapes]
    blob_h = torch.randn(sum(sizes), dtype=torch.bfloat16).pin_memory()
    blob_d = torch.empty_like(blob_h, device="cuda")
    dev, off = {}, 0
    for (key, sh), n in zip(shapes, sizes):       # views of the device blob
        dev[key] = blob_d[off:off + n].view(*sh)
        off += n
    stream = torch.cuda.current_stream()
    times = []
    nbytes = blob_h.numel() * 2
    for it in range(60):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        blob_d.copy_(blob_h, non_blocking=True)
        for li in range(w.n_layers):
            A = {p: dev[(li, p, "A")] for p in w.lora_targets}
            Bf = {p: dev[(li, p, "B")] for p in w.lora_targets}
            B.vfm_lora_attach(model.lora[li], t, r, w.lora_scale, A, Bf, stream)
        B.vfm_head_attach(model.head_tab, t, n_out, dev[("head", "W")], dev[("head", "b")], stream=stream)
        torch.cuda.synchronize()
        if it >= 10:
            times.append(time.perf_counter() - t0)
    ms = float(np.median(times)) * 1e3
    print(json.dumps({"metric": "task load time (LoRA factors of every layer + head, host to attached)",
                      "value": ms, "unit": "ms", "higher_is_better": False, "n_gpus": 1,
                      "config": {"workload": w.name, "layers": w.n_layers, "lora_rank": r,
                                 "lora_targets": list(w.lora_targets), "head_outputs": n_out,
                                 "bytes": int(nbytes)},
                      "loads_timed": len(times)}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=4,
                    help="1 tiny fp32 encoder, 2 ViT-B, 3 time-series encoder, "
                         "4 7B decoder prefill (default), 5 7B decoder decode")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--task-load", action="store_true",
                    help="time loading one task's adapters and head into the ViT-B-shaped backbone")
    ap.add_argument("--loop", type=int, default=0,
                    help="run the continuous-batching loop over this many requests instead of one step")
    ap.add_argument("--admission", choices=("fifo", "bfq"), default="fifo",
                    help="--loop: admit prompts FIFO or by BFQ (16-request batches, decode tokens charged)")
    ap.add_argument("--paged", type=int, default=0,
                    help="decode workloads: read the KV cache through pages of this many slots "
                         "(random page order) instead of the contiguous cache")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}): the mixed-task forward "
              "shards by request with no cross-GPU exchange, and bench.py measures one GPU's "
              "share.", file=sys.stderr)
        sys.exit(2)

    if args.loop:
        loop_bench(args)
        return
    if args.task_load:
        task_load_bench(args)
        return

    import torch
    from paper_2606_09643_amd import binding as B
    from paper_2606_09643_amd import runner as R
    from paper_2606_09643_amd import workloads as wl

    w = wl.WORKLOADS[args.workload]
    batch = wl.draw_batch(w)
    model = R.Model(w)
    inp = R.Inputs(w, batch)
    kv = R.KVCache(w, batch, w.n_layers) if w.mode == "decode" else None
    pb = R.make_batch(w, batch, model.heads, kv)
    fwd = R.Forward(model, pb, inp, kv)
    if args.paged:
        if kv is None:
            print("--paged applies to decode workloads only", file=sys.stderr)
            sys.exit(2)
        fwd.paged = R.page_kv_cache(kv, batch, args.paged)
        torch.cuda.empty_cache()
    ranks = wl.task_ranks(w)
    work = algorithmic_work(w, batch, ranks, model.heads.n_out if model.heads is not None else None)
    stream = torch.cuda.current_stream()

    # Calibration for HBM-traffic counters: one plain device copy of a known
    # size (256 MiB read + 256 MiB written), outside the timed region.
    cal_src = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
    cal_dst = torch.empty_like(cal_src)
    cal_dst.copy_(cal_src)
    torch.cuda.synchronize()
    del cal_src, cal_dst

    for _ in range(args.warmup):
        fwd(stream)
    torch.cuda.synchronize()

    # Timed region: exactly `steps` forwards, each bracketed by its own pair
    # of events on the forward's stream; the dominant kernel class is timed
    # with hipEvents around each of its launches inside the same region (the
    # library records them on the stream it launches on).
    dom = "attn" if w.mode == "decode" else "gemm_up"
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    torch.cuda.synchronize()
    B.vfm_profile_enable([dom])
    t_wall = time.perf_counter()
    for e0, e1 in ev:
        e0.record(stream)
        fwd(stream)
        e1.record(stream)
    torch.cuda.synchronize()
    wall_s = time.perf_counter() - t_wall
    prof = B.vfm_profile_read()
    B.vfm_profile_enable([])
    step_ms = np.array([e0.elapsed_time(e1) for e0, e1 in ev])
    ms_step = float(np.median(step_ms))
    tokens = batch.total_rows
    value = tokens / (ms_step * 1e-3)

    dom_ms, dom_n = prof[dom]
    avg_ms = dom_ms / max(dom_n, 1)
    if w.mode == "decode":
        per_launch = work["kv_read_bytes_per_layer"]
        achieved = per_launch / (avg_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": achieved / PEAK_HBM_GBS, "traffic": None}
    else:
        per_launch = work["per_launch_flops"][dom]
        peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_FP32_TFLOPS
        achieved = per_launch / (avg_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                "frac": achieved / peak, "traffic": None}
    roof["traffic"] = hbm_traffic(w.name, dom)
    if dom == "attn":
        kname = "attn_decode_kernel (KV-cache attention" + (f", pages of {args.paged})" if args.paged else ")")
    elif w.dtype != "bf16":
        kname = "gemm_f32_kernel (MLP up projection + GELU)"
    elif w.family == "decoder":
        kname = "gemm_bf16_large_kernel (gate/up projections + SwiGLU" + (
            ", LoRA fused)" if {"gate", "up"} & set(w.lora_targets) else ")")
    else:
        kname = "gemm_bf16_large_kernel (MLP up projection + GELU" + (
            ", LoRA fused)" if "up" in w.lora_targets else ")")
    roof.update({"kernel": kname,
                 "avg_launch_ms": avg_ms, "launches": dom_n, "per_launch": per_launch})

    step_tflops = work["step_flops"] / (ms_step * 1e-3) / 1e12
    peak_step = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_FP32_TFLOPS
    out = {
        "metric": METRIC, "value": value, "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32", "data": "synthetic",
        "config": {"workload": w.name, "n_req": w.n_req, "tokens": tokens,
                   "n_tasks": w.n_tasks, "distinct_tasks": int(len(np.unique(batch.task_id))),
                   "layers": w.n_layers, "d_model": w.d, "d_ff": w.d_ff, "lora_rank": w.rank,
                   "lora_targets": list(w.lora_targets),
                   "kv_cache": f"paged {args.paged}" if args.paged else "contiguous"},
        "ms_per_step_mean": float(step_ms.mean()), "ms_per_step_min": float(step_ms.min()),
        "ms_per_step_max": float(step_ms.max()), "timed_wall_s": wall_s,
        "step_tflops": step_tflops,
        "step_roofline_frac": step_tflops / peak_step if w.mode != "decode" else
        (work["step_bytes"] / (ms_step * 1e-3) / 1e9) / PEAK_HBM_GBS,
        "roofline": roof,
    }
    if args.paged:
        roof["traffic"] = None          # counters were taken on the contiguous cache
    if not args.no_cpu_baseline and not args.paged:
        out["cpu_baseline"] = cpu_baseline(w, batch, model, inp, kv)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
