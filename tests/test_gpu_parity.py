"""GPU parity of the HIP path against the fp64 oracle, call by call.

Every case feeds the oracle exactly the tensors the GPU received (the GPU
layer's own input rows are downloaded before each layer), and compares with
the row-normwise relative error (max over rows of max|g - o| / max|o|):
2e-2 for bf16 workloads, 1e-5 for the fp32 one.  Integer plan outputs are
checked bit-exact on the host (tests/test_abi_cpu.py).
"""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import vfm_oracle as O
from paper_2606_09643_amd import binding as B
from paper_2606_09643_amd import runner as R
from paper_2606_09643_amd import workloads as wl
from tests.gpu_common import (as_f32, expected_embed, log, oracle_heads, oracle_layer_rows, oracle_plan,
                               seeded_rows, set_rows,
                              pick_requests, tol)
from tests.helpers import np64, oracle_adapter, oracle_weights, spec_of

pytestmark = pytest.mark.gpu


def _batch(w, task_id, seq_len, ctx=None):
    return wl.Batch(np.asarray(task_id, np.int32), np.asarray(seq_len, np.int32),
                    None if ctx is None else np.asarray(ctx, np.int32))


# Small cases per workload: real widths, few requests, ragged lengths.
SMALL = {
    1: dict(task_id=[3, 0, 1, 1, 2, 0, 3, 2], seq_len=[64] * 8),
    2: dict(task_id=[5, 0, 5, 2, 9, 0], seq_len=[197] * 6),
    3: dict(task_id=[1, 1, 7, 0, 31, 7], seq_len=[64] * 6),
    4: dict(task_id=[3, 0, 3, 63], seq_len=[1, 130, 64, 77]),
    5: dict(task_id=[2, 2, 0, 127, 5], seq_len=[1] * 5, ctx=[0, 63, 300, 64, 4200]),
}


def _setup(idx, n_layers=1, b_std=0.01, ranks=None, case=None):
    w = wl.WORKLOADS[idx]
    case = case or SMALL[idx]
    batch = _batch(w, **case)
    model = R.Model(w, n_layers=n_layers, b_std=b_std, ranks=ranks)
    inp = R.Inputs(w, batch)
    kv = R.KVCache(w, batch, n_layers) if w.mode == "decode" else None
    pb = R.make_batch(w, batch, model.heads, kv)
    fwd = R.Forward(model, pb, inp, kv)
    pl = oracle_plan(w, batch, model.heads.n_out if model.heads is not None else None)
    return w, batch, model, inp, kv, pb, fwd, pl


@pytest.mark.parametrize("idx", [1, 2, 3, 4, 5])
def test_embed_exact(idx):
    w, batch, model, inp, kv, pb, fwd, pl = _setup(idx)
    log(f"embed workload {idx} T={pb.T}")
    fwd.embed()
    torch.cuda.synchronize()
    got = fwd.x.double().cpu().numpy()
    ref = expected_embed(w, batch, inp, pl)
    if inp.mode == B.VFM_EMBED_PATCHES:
        assert O.row_rel_error(got, ref) < 1e-5
    else:
        assert np.array_equal(got, ref)


# b_std 0.1 makes the adapters' difference about as large as the shared
# projection itself (std ~0.8 vs ~1), so a LoRA slip cannot hide under the
# tolerance; much larger factors (0.3) push the attention logits' spread to
# ~7 where the bf16 rounding of q and k alone moves outputs by ~3%.
@pytest.mark.parametrize("idx,b_std", [(1, 0.01), (1, 0.3), (2, 0.01), (2, 0.1), (3, 0.01),
                                       (3, 0.1), (4, 0.01), (4, 0.1), (5, 0.01), (5, 0.1)])
def test_layer_parity(idx, b_std):
    ranks = None
    if b_std > 0.01:  # strong adapters, mixed ranks incl. zero
        w = wl.WORKLOADS[idx]
        ranks = np.array([(8 * (t % 3)) for t in range(w.n_tasks)], np.int32)
        ranks[ranks == 0] = 0
    w, batch, model, inp, kv, pb, fwd, pl = _setup(idx, n_layers=1, b_std=b_std, ranks=ranks)
    log(f"layer workload {idx} b_std={b_std} T={pb.T}")
    x_in = as_f32(expected_embed(w, batch, inp, pl))
    set_rows(fwd.x, x_in)
    fwd.layer(0)
    torch.cuda.synchronize()
    got = fwd.x.double().cpu().numpy()
    W_np = oracle_weights(model.layers[0])
    reqs = list(range(batch.n_req))
    res = oracle_layer_rows(w, W_np, model.adapters[0], pl, x_in, reqs, kv=kv, li=0)
    cu = pl["cu_seqlens"]
    worst = 0.0
    for p in reqs:
        e = O.row_rel_error(got[cu[p]:cu[p + 1]], res[p][0])
        worst = max(worst, e)
    log(f"  max row rel err {worst:.3e}")
    assert worst < tol(w)
    if kv is not None:  # the new K / V rows landed in their slots
        for p in reqs:
            i = int(pl["order"][p])
            slot = int(kv.kv_start[i] + batch.ctx[i])
            kr, vr = kv.rows(0, slot, 1)
            kg = kr.double().cpu().numpy()
            vg = vr.double().cpu().numpy()
            assert O.row_rel_error(kg, res[p][1]) < tol(w)
            assert O.row_rel_error(vg, res[p][2]) < tol(w)


@pytest.mark.parametrize("idx", [1, 2, 3, 5])
def test_head_parity(idx):
    w, batch, model, inp, kv, pb, fwd, pl = _setup(idx)
    log(f"head workload {idx}")
    x_plan = seeded_rows(pb.T, w.d, 100 + idx)
    set_rows(fwd.x, x_plan)
    fwd.head()
    torch.cuda.synchronize()
    got = fwd.out.cpu().numpy()
    ref = oracle_heads(w, model, pl, x_plan, model.heads.n_out)
    off = pl["logit_off"]
    worst = max(O.row_rel_error(got[off[i]:off[i + 1]][None], ref[i][None]) for i in range(batch.n_req))
    log(f"  max rel err {worst:.3e}")
    assert worst < tol(w)


def test_final_hidden_unpermuted():
    """Decoder prefill returns the final-normed rows in original order."""
    w, batch, model, inp, kv, pb, fwd, pl = _setup(4)
    x_plan = as_f32(expected_embed(w, batch, inp, pl))
    set_rows(fwd.x, x_plan)
    fwd.head()
    torch.cuda.synchronize()
    got = fwd.out.double().cpu().numpy()
    cu, cu_o = pl["cu_seqlens"], pl["cu_orig"]
    fw = np64(model.final["w"])
    for p, i in enumerate(pl["order"]):
        ref = O.rms_norm(x_plan[cu[p]:cu[p + 1]], fw, w.norm_eps)
        assert O.row_rel_error(got[cu_o[i]:cu_o[i + 1]], ref) < tol(w)


@pytest.mark.parametrize("dtype,idx", [("f32", 1), ("bf16", 2), ("bf16", 5)])
def test_lora_apply(dtype, idx):
    """vfm_lora_apply alone: y += s_t (x A_t^T) B_t^T per task segment,
    ranks 0 / 8 / 16 / 64 mixed."""
    w = wl.WORKLOADS[idx]
    n_tasks = 6
    w = w.replace(n_tasks=n_tasks)
    ranks = np.array([0, 8, 16, 64, 8, 0], np.int32)
    ad = wl.adapters_layer(w, 0, device="cuda", ranks=ranks, b_std=0.1, targets=("q", "down"))
    tab = R.lora_table(w, ad)
    r = np.random.default_rng(3)
    task_id = r.integers(0, n_tasks, size=23)
    seq_len = r.integers(1, 90, size=23)
    pb = B.Batch(task_id, seq_len, n_tasks)
    pl = O.plan(task_id, seq_len, n_tasks)
    for proj in ("q", "down"):
        d_in, d_out = wl.proj_dims(w, proj)
        x = torch.randn(pb.T, d_in, device="cuda").to(w.torch_dtype)
        y0 = torch.randn(pb.T, d_out, device="cuda")
        y = y0.clone()
        ws = torch.empty(pb.T * 64 * 4 + 4096, dtype=torch.uint8, device="cuda")
        B.vfm_lora_apply(B.VFM_BF16 if dtype == "bf16" else B.VFM_F32, wl.PROJ_INDEX[proj], d_in,
                         d_out, tab.c, pb.c, x, y, ws)
        torch.cuda.synchronize()
        delta = (y - y0).double().cpu().numpy()
        xn = np64(x)
        worst = 0.0
        for t in range(n_tasks):
            r0, r1 = int(pl["seg_row"][t]), int(pl["seg_row"][t + 1])
            if r1 == r0:
                continue
            if ranks[t] == 0:
                assert np.array_equal(y[r0:r1].cpu().numpy(), y0[r0:r1].cpu().numpy())
                continue
            ref = O.lora_delta(xn[r0:r1], np64(ad.a(proj, t)), np64(ad.b(proj, t)), float(ad.scale[t]))
            worst = max(worst, O.row_rel_error(delta[r0:r1], ref))
        log(f"lora_apply {dtype} {proj} max rel err {worst:.3e}")
        assert worst < (2e-2 if dtype == "bf16" else 1e-5)


# Batch-invariance cases: workload 2 with every task alone still above the
# small-batch threshold (large-tile kernels), workload 4 below it (split-K).
# The "tail" cases make the large-tile GEMMs compute a task's rows with other
# tile shapes than when the task runs alone: the mixed batch's last,
# partly filled round of 256 x 256 tiles goes to a second launch of 256 x 128
# tiles (7B O / down: rows 4096.. of 5300; ViT-B MLP-up: rows 5376.. of
# 7092), while alone the first task's O / down (1204 rows, workload 4) and
# QKV (2758 rows, workload 2) run as 256 x 128 and the other tasks' rows as
# 256 x 256 tiles; both also cross the row count at which the pre-norms of
# the old code switched kernels.  "4-mixlen" puts 200-row prompts (the
# whole-request attention kernel) beside 300-row ones (the flash kernel).
INVARIANCE = {
    "2": (2, dict(task_id=[5, 0, 2, 0, 5, 2, 2, 5, 0, 5, 0, 2, 0, 2, 5, 5, 2, 0], seq_len=[197] * 18)),
    "4": (4, SMALL[4]),
    "2-tail": (2, dict(task_id=[0] * 14 + [5] * 14 + [9] * 8, seq_len=[197] * 36)),
    "4-tail": (4, dict(task_id=[1, 1, 9, 9, 9, 9], seq_len=[602, 602, 1024, 1024, 1024, 1024])),
    "4-mixlen": (4, dict(task_id=[1] * 6 + [9] * 4, seq_len=[200] * 6 + [300] * 4)),
    # 17 000 rows: more 64-row tiles than CUs, so the large-batch LoRA shrink
    # takes 96-row tiles, while each task alone (12 000 / 5 000 rows) keeps
    # the plan's 64-row tiles
    "4-big": (4, dict(task_id=[1] * 12 + [9] * 5, seq_len=[1000] * 17)),
    # larger ranks take the unpacked LoRA steps of the large GEMM: half
    # steps (rank <= 32) and, above 32, two steps per SwiGLU run
    "2-tail-r32": (2, dict(task_id=[0] * 14 + [5] * 14 + [9] * 8, seq_len=[197] * 36), 32),
    "4-tail-r64": (4, dict(task_id=[1, 1, 9, 9, 9, 9], seq_len=[602, 602, 1024, 1024, 1024, 1024]), 64),
}


@pytest.mark.parametrize("name", list(INVARIANCE))
def test_batch_invariance_and_zero_rank_bit_exact(name):
    """A task's rows are bit-identical whether co-batched with other tasks or
    run alone (both batches on one side of the small-batch threshold), and a
    rank-0 task equals the bare backbone bit for bit."""
    idx, case, *rank = INVARIANCE[name]
    w = wl.WORKLOADS[idx]
    ranks = np.full(w.n_tasks, rank[0] if rank else w.rank, np.int32)
    ranks[0] = 0
    w_, batch, model, inp, kv, pb, fwd, pl = _setup(idx, n_layers=1, ranks=ranks, b_std=0.1,
                                                    case=case)
    small = pb.T < B.VFM_SMALL_BATCH_ROWS
    fwd.embed()
    fwd.layer(0)
    torch.cuda.synchronize()
    mixed = fwd.x.cpu().numpy()
    src = inp.src
    for t in sorted(set(case["task_id"])):
        keep = [i for i, tt in enumerate(case["task_id"]) if tt == t]
        sub = _batch(w, [case["task_id"][i] for i in keep], [case["seq_len"][i] for i in keep])
        pbs = R.make_batch(w, sub, model.heads)
        assert (pbs.T < B.VFM_SMALL_BATCH_ROWS) == small
        inps = R.Inputs(w, sub)
        # the same input rows as in the mixed batch
        cu_o = pl["cu_orig"]
        if inp.mode == B.VFM_EMBED_ROWS:
            inps.src = torch.cat([src[cu_o[i]:cu_o[i + 1]] for i in keep])
        else:
            inps.src = torch.cat([src[cu_o[i]:cu_o[i + 1]] for i in keep])
            inps.table = inp.table
        f2 = R.Forward(model, pbs, inps)
        f2.embed()
        f2.layer(0)
        torch.cuda.synchronize()
        alone = f2.x.cpu().numpy()
        seg = slice(int(pl["seg_row"][t]), int(pl["seg_row"][t + 1]))
        assert np.array_equal(mixed[seg], alone), f"task {t}"
        if t == 0:  # rank 0: equals the backbone with no adapters at all
            bare = R.Model(w, n_layers=1, with_lora=False)
            f3 = R.Forward(bare, pbs, inps)
            f3.embed()
            f3.layer(0)
            torch.cuda.synchronize()
            assert np.array_equal(f3.x.cpu().numpy(), alone)


def test_merged_weights_match_adapter_path():
    """Running the bare path on W + s B A (merged in fp32, rounded once) agrees
    with the unmerged per-task path for a batch of one task."""
    w = wl.WORKLOADS[2]
    case = dict(task_id=[5, 5], seq_len=[197, 197])
    w_, batch, model, inp, kv, pb, fwd, pl = _setup(2, n_layers=1, b_std=0.1, case=case)
    fwd.embed()
    fwd.layer(0)
    torch.cuda.synchronize()
    got = fwd.x.double().cpu().numpy()
    bare = R.Model(w, n_layers=1, with_lora=False)
    W = bare.layers[0]
    ad = model.adapters[0]
    d = w.d
    t = 5
    with torch.no_grad():
        for p, (lo, hi) in (("q", (0, d)), ("k", (d, 2 * d)), ("v", (2 * d, 3 * d))):
            m = W["w_qkv"][lo:hi].float() + float(ad.scale[t]) * (ad.b(p, t).float() @ ad.a(p, t).float())
            W["w_qkv"][lo:hi] = m.to(W["w_qkv"].dtype)
        W["w_o"].copy_((W["w_o"].float() + float(ad.scale[t]) * (ad.b("o", t).float() @ ad.a("o", t).float())).to(W["w_o"].dtype))
    bare.c_layers[0] = B.layer_weights(W)
    f2 = R.Forward(bare, pb, inp)
    f2.embed()
    f2.layer(0)
    torch.cuda.synchronize()
    assert O.row_rel_error(f2.x.double().cpu().numpy(), got) < tol(w)


@pytest.mark.parametrize("idx", [1, 2, 3])
def test_end_to_end_small(idx):
    """All layers + head from the initial input against the oracle chain."""
    w = wl.WORKLOADS[idx]
    n_layers = w.n_layers if idx != 3 else 6
    w_, batch, model, inp, kv, pb, fwd, pl = _setup(idx, n_layers=n_layers)
    log(f"end-to-end workload {idx} layers={n_layers}")
    out = fwd().cpu().numpy()
    torch.cuda.synchronize()
    x = expected_embed(w, batch, inp, pl)
    cu = pl["cu_seqlens"]
    for li in range(n_layers):
        W_np = oracle_weights(model.layers[li])
        res = oracle_layer_rows(w, W_np, model.adapters[li], pl, x, range(batch.n_req))
        x = np.concatenate([res[p][0] for p in range(batch.n_req)])
    ref = oracle_heads(w, model, pl, x, model.heads.n_out)
    off = pl["logit_off"]
    worst = max(O.row_rel_error(out[off[i]:off[i + 1]][None], ref[i][None]) for i in range(batch.n_req))
    log(f"  end-to-end logits max rel err {worst:.3e}")
    assert worst < tol(w)


def test_bench_workload_full_size_sampled():
    """The benchmarked workload (ViT-B-shaped, 64 requests x 197 tokens,
    16 tasks, 12 layers) in the bench's launch configuration: every layer's
    output on sampled requests against the oracle, both sides starting each
    layer from the oracle's rows, and those requests' head outputs."""
    w = wl.WORKLOADS[2]
    batch = wl.draw_batch(w)
    model = R.Model(w)
    inp = R.Inputs(w, batch)
    pb = R.make_batch(w, batch, model.heads)
    fwd = R.Forward(model, pb, inp)
    pl = oracle_plan(w, batch, model.heads.n_out)
    reqs = pick_requests(pl)
    log(f"full-size bench workload, sampled plan positions {reqs}")
    x_or = as_f32(expected_embed(w, batch, inp, pl))
    set_rows(fwd.x, x_or)
    cu = pl["cu_seqlens"]
    worst = 0.0
    for li in range(w.n_layers):
        res = oracle_layer_rows(w, oracle_weights(model.layers[li]), model.adapters[li], pl, x_or, reqs)
        fwd.layer(li)
        torch.cuda.synchronize()
        got = fwd.x.double().cpu().numpy()
        for p in reqs:
            worst = max(worst, O.row_rel_error(got[cu[p]:cu[p + 1]], res[p][0]))
            # both sides take the oracle's rows into the next layer
            x_or[cu[p]:cu[p + 1]] = as_f32(res[p][0])
            set_rows(fwd.x, x_or[cu[p]:cu[p + 1]], int(cu[p]))
    log(f"  per-layer max row rel err {worst:.3e}")
    assert worst < tol(w)
    fwd.head()
    torch.cuda.synchronize()
    out = fwd.out.cpu().numpy()
    ref = oracle_heads(w, model, pl, x_or, model.heads.n_out)
    off = pl["logit_off"]
    hw = max(O.row_rel_error(out[off[i]:off[i + 1]][None], ref[i][None])
             for i in (int(pl["order"][p]) for p in reqs))
    log(f"  head max rel err {hw:.3e}")
    assert hw < tol(w)


def test_layer_parity_long_prompts():
    """Causal prompts longer than 256 tokens take the flash (online-softmax)
    attention kernel: ragged 300 / 1 / 513-token prompts, 0.1 adapters."""
    case = dict(task_id=[3, 0, 63], seq_len=[300, 1, 513])
    w, batch, model, inp, kv, pb, fwd, pl = _setup(4, n_layers=1, b_std=0.1, case=case)
    log(f"layer workload 4 long prompts T={pb.T}")
    x_in = as_f32(expected_embed(w, batch, inp, pl))
    set_rows(fwd.x, x_in)
    fwd.layer(0)
    torch.cuda.synchronize()
    got = fwd.x.double().cpu().numpy()
    res = oracle_layer_rows(w, oracle_weights(model.layers[0]), model.adapters[0], pl, x_in,
                            range(batch.n_req))
    cu = pl["cu_seqlens"]
    worst = max(O.row_rel_error(got[cu[p]:cu[p + 1]], res[p][0]) for p in range(batch.n_req))
    log(f"  max row rel err {worst:.3e}")
    assert worst < tol(w)


def test_large_gemm_many_task_runs():
    """Large-batch projections (T >= 1024 rows) where each 256-row tile holds
    many short requests of different tasks, with task ids absent from the
    batch between them and ranks 0 / 8 / 16 mixed: the tile's LoRA steps
    must visit exactly the task runs present (up to ~20 per tile here) and
    no others.  Decoder layer, 0.1 adapters, every request checked."""
    rng = np.random.default_rng(7)
    n = 96
    present = np.sort(rng.choice(64, size=40, replace=False))   # 24 task ids absent
    task_id = rng.choice(present, size=n)
    seq_len = 1 + (np.arange(n) * 7) % 25
    ranks = np.array([8 * (t % 3) for t in range(64)], np.int32)
    case = dict(task_id=task_id.tolist(), seq_len=seq_len.tolist())
    w, batch, model, inp, kv, pb, fwd, pl = _setup(4, n_layers=1, b_std=0.1, ranks=ranks, case=case)
    assert pb.T >= 1024, pb.T                      # the large-tile GEMM path
    log(f"layer workload 4, {n} short requests over {len(present)} tasks, T={pb.T}")
    x_in = as_f32(expected_embed(w, batch, inp, pl))
    set_rows(fwd.x, x_in)
    fwd.layer(0)
    torch.cuda.synchronize()
    got = fwd.x.double().cpu().numpy()
    res = oracle_layer_rows(w, oracle_weights(model.layers[0]), model.adapters[0], pl, x_in,
                            range(batch.n_req))
    cu = pl["cu_seqlens"]
    worst = max(O.row_rel_error(got[cu[p]:cu[p + 1]], res[p][0]) for p in range(batch.n_req))
    log(f"  max row rel err {worst:.3e}")
    assert worst < tol(w)


@pytest.mark.parametrize("ranks", [(0, 8, 24, 32), (16, 40, 64, 8)])
def test_large_gemm_ranks_above_16(ranks):
    """The large GEMM's LoRA steps for ranks above 16 (one run per step:
    half steps up to rank 32, and above 32 a SwiGLU run's gate and up
    steps), over short requests of many tasks as in the test above.  B's
    spread is scaled by sqrt(16 / largest rank), so the adapters' difference
    has the size of a rank-16 adapter with B ~ N(0, 0.1), the strength the
    bf16 tolerance is set for (a rank-r difference grows as sqrt(r))."""
    b_std = 0.1 * np.sqrt(16 / max(ranks))
    rng = np.random.default_rng(11)
    n = 96
    task_id = rng.integers(0, 64, size=n)
    seq_len = 1 + (np.arange(n) * 7) % 25
    rk = np.array([ranks[t % len(ranks)] for t in range(64)], np.int32)
    case = dict(task_id=task_id.tolist(), seq_len=seq_len.tolist())
    w, batch, model, inp, kv, pb, fwd, pl = _setup(4, n_layers=1, b_std=b_std, ranks=rk, case=case)
    assert pb.T >= 1024, pb.T
    log(f"layer workload 4, ranks {ranks}, B ~ N(0, {b_std:.3f}), {n} short requests, T={pb.T}")
    x_in = as_f32(expected_embed(w, batch, inp, pl))
    set_rows(fwd.x, x_in)
    fwd.layer(0)
    torch.cuda.synchronize()
    got = fwd.x.double().cpu().numpy()
    res = oracle_layer_rows(w, oracle_weights(model.layers[0]), model.adapters[0], pl, x_in,
                            range(batch.n_req))
    cu = pl["cu_seqlens"]
    worst = max(O.row_rel_error(got[cu[p]:cu[p + 1]], res[p][0]) for p in range(batch.n_req))
    log(f"  max row rel err {worst:.3e}")
    assert worst < tol(w)


def test_packed_lora_steps_bit_exact():
    """Runs of a tile share a LoRA step (up to four of rank <= 16): a task
    whose rows sit among many one-row requests of other tasks (so its run
    shares steps with theirs, in another slot than when alone) gives the
    same bits as the task run alone, and matches the oracle; the one-row
    requests match the oracle too."""
    w = wl.WORKLOADS[4]
    big = 9
    singles_lo = list(range(1, 8))                  # its run is the eighth of the first tile
    singles_hi = list(range(10, 51))                # 41 one-row runs after its last rows
    task_id = singles_lo + [big] * 3 + singles_hi
    seq_len = [1] * len(singles_lo) + [400] * 3 + [1] * len(singles_hi)
    ranks = np.array([8 * (t % 3) for t in range(w.n_tasks)], np.int32)
    ranks[big] = 16
    case = dict(task_id=task_id, seq_len=seq_len)
    w, batch, model, inp, kv, pb, fwd, pl = _setup(4, n_layers=1, b_std=0.1, ranks=ranks, case=case)
    assert pb.T >= B.VFM_SMALL_BATCH_ROWS
    log(f"layer workload 4, task {big} (1200 rows) among {len(singles_lo) + len(singles_hi)} one-row tasks")
    x_in = as_f32(expected_embed(w, batch, inp, pl))
    set_rows(fwd.x, x_in)
    fwd.layer(0)
    torch.cuda.synchronize()
    mixed = fwd.x.cpu().numpy()
    res = oracle_layer_rows(w, oracle_weights(model.layers[0]), model.adapters[0], pl, x_in,
                            range(batch.n_req))
    cu = pl["cu_seqlens"]
    worst = max(O.row_rel_error(mixed[cu[p]:cu[p + 1]].astype(np.float64), res[p][0])
                for p in range(batch.n_req))
    log(f"  max row rel err {worst:.3e}")
    assert worst < tol(w)
    # the task alone: its requests in the same order, so its plan rows are
    # the mixed plan's segment of that task
    keep = [i for i, t in enumerate(task_id) if t == big]
    sub = _batch(w, [big] * len(keep), [seq_len[i] for i in keep])
    pbs = R.make_batch(w, sub, model.heads)
    assert pbs.T >= B.VFM_SMALL_BATCH_ROWS
    f2 = R.Forward(model, pbs, R.Inputs(w, sub))
    seg = slice(int(pl["seg_row"][big]), int(pl["seg_row"][big + 1]))
    set_rows(f2.x, x_in[seg])
    f2.layer(0)
    torch.cuda.synchronize()
    assert np.array_equal(mixed[seg], f2.x.cpu().numpy())


@pytest.mark.parametrize("idx", [1, 3, 4, 5])
def test_full_size_sampled(idx):
    """Each remaining workload at its full batch, in the bench's launch
    configuration: every layer's output on sampled requests against the
    oracle, both sides starting each layer from the oracle's rows (parity
    call by call, through all 24 / 32 layers), and those requests' head
    outputs; decode also checks the new K / V rows written to the cache."""
    w = wl.WORKLOADS[idx]
    n_layers = w.n_layers
    batch = wl.draw_batch(w)
    model = R.Model(w, n_layers=n_layers)
    inp = R.Inputs(w, batch)
    kv = R.KVCache(w, batch, n_layers) if w.mode == "decode" else None
    pb = R.make_batch(w, batch, model.heads, kv)
    fwd = R.Forward(model, pb, inp, kv)
    pl = oracle_plan(w, batch, model.heads.n_out if model.heads is not None else None)
    if idx == 4:      # the shortest prompt and a 300..512-token one at a task boundary (oracle cost)
        lens = np.diff(pl["cu_seqlens"])
        seg = pl["seg_req"]
        bound = sorted({int(seg[t]) for t in range(w.n_tasks) if seg[t + 1] > seg[t]} |
                       {int(seg[t + 1]) - 1 for t in range(w.n_tasks) if seg[t + 1] > seg[t]})
        mid = [p for p in bound if 300 <= lens[p] <= 512] or [int(np.argsort(lens)[len(lens) // 2])]
        reqs = [int(np.argmin(lens)), mid[0]]
    else:
        reqs = pick_requests(pl, k=6)
    log(f"full-size workload {idx}: T={pb.T}, {n_layers} layers, sampled plan positions {reqs}")
    x_or = as_f32(expected_embed(w, batch, inp, pl))
    set_rows(fwd.x, x_or)
    cu = pl["cu_seqlens"]
    worst = 0.0
    for li in range(n_layers):
        res = oracle_layer_rows(w, oracle_weights(model.layers[li]), model.adapters[li], pl, x_or, reqs,
                                kv=kv, li=li)
        fwd.layer(li)
        torch.cuda.synchronize()
        got = fwd.x.double().cpu().numpy()
        for p in reqs:
            worst = max(worst, O.row_rel_error(got[cu[p]:cu[p + 1]], res[p][0]))
            # both sides take the oracle's rows into the next layer
            x_or[cu[p]:cu[p + 1]] = as_f32(res[p][0])
            set_rows(fwd.x, x_or[cu[p]:cu[p + 1]], int(cu[p]))
            if kv is not None:
                i = int(pl["order"][p])
                slot = int(kv.kv_start[i] + batch.ctx[i])
                kr, vr = kv.rows(li, slot, 1)
                assert O.row_rel_error(kr.double().cpu().numpy(), res[p][1]) < tol(w)
                assert O.row_rel_error(vr.double().cpu().numpy(), res[p][2]) < tol(w)
        log(f"  layer {li}: max row rel err so far {worst:.3e}")
    assert worst < tol(w)
    if model.heads is not None and n_layers == w.n_layers:
        fwd.head()
        torch.cuda.synchronize()
        out = fwd.out.cpu().numpy()
        ref = oracle_heads(w, model, pl, x_or, model.heads.n_out)
        off = pl["logit_off"]
        hw = max(O.row_rel_error(out[off[i]:off[i + 1]][None], ref[i][None])
                 for i in (int(pl["order"][p]) for p in reqs))
        log(f"  head max rel err {hw:.3e}")
        assert hw < tol(w)


@pytest.mark.parametrize("rope", [True, False])
def test_prefill_writes_kv_cache(rope):
    """A causal (prefill) layer given a KV cache writes each row's rotated
    key and its value at slot kv_start + pos of every head of the head-major
    cache: with RoPE the rotation pass writes them, without it the cache-write
    kernel does.  Slots between the requests keep their previous contents.
    Decoder layer, ragged prompts (1, 130, 64, 77 tokens)."""
    _prefill_with_cache(wl.WORKLOADS[4], SMALL[4], rope)


@pytest.mark.parametrize("hd", [64, 128])
def test_large_batch_rope_in_gemm_with_cache(hd):
    """A batch above the small-batch threshold on a decoder of width 1024
    with head_dim 64 or 128: the QKV GEMM's store pass applies RoPE (tiles
    holding whole heads) and the cache-write kernel copies the rotated keys
    and the values to the cache.  Outputs and cached K / V against the
    oracle, gap slots untouched; ragged prompts of 300, 1, 513 and 260."""
    w = dataclasses.replace(wl.WORKLOADS[4], d=1024, n_heads=1024 // hd, head_dim=hd, d_ff=2816, n_tasks=8)
    case = dict(task_id=[3, 0, 7, 3], seq_len=[300, 1, 513, 260])
    assert sum(case["seq_len"]) >= B.VFM_SMALL_BATCH_ROWS
    _prefill_with_cache(w, case, True)


def _prefill_with_cache(w, case, rope):
    batch = _batch(w, **case)
    model = R.Model(w, n_layers=1, b_std=0.1)
    inp = R.Inputs(w, batch)
    gap = 3
    lens = batch.seq_len.astype(np.int64)
    kvs = np.zeros(batch.n_req, np.int64)
    kvs[1:] = np.cumsum(lens + gap)[:-1]
    slots = int((lens + gap).sum())
    pb = B.Batch(batch.task_id, batch.seq_len, w.n_tasks, ctx_len=np.zeros(batch.n_req, np.int32),
                 kv_start=kvs.astype(np.int32))
    fwd = R.Forward(model, pb, inp)
    cfg = R.cfg_for(w)
    if not rope:
        cfg.rope_theta = 0.0
    sentinel = 7.0
    kc = torch.full((w.n_heads, slots, w.head_dim), sentinel, dtype=torch.bfloat16, device="cuda")
    vc = torch.full_like(kc, sentinel)
    log(f"prefill layer with KV cache, d={w.d}, head_dim={w.head_dim}, rope={rope}, T={pb.T}, slots={slots}")
    pl = oracle_plan(w, batch)
    x_in = as_f32(expected_embed(w, batch, inp, pl))
    set_rows(fwd.x, x_in)
    B.vfm_layer_forward(cfg, model.c_layers[0], model.lora_c(0), pb.c, fwd.x, kc, vc, slots, fwd.ws)
    torch.cuda.synchronize()
    got = fwd.x.double().cpu().numpy()
    spec = spec_of(w)
    if not rope:
        spec["rope_theta"] = 0.0
    cu = pl["cu_seqlens"]
    W_np = oracle_weights(model.layers[0])
    k_all = kc.permute(1, 0, 2).reshape(slots, w.d).double().cpu().numpy()
    v_all = vc.permute(1, 0, 2).reshape(slots, w.d).double().cpu().numpy()
    written = np.zeros(slots, bool)
    worst = 0.0
    for p in range(batch.n_req):
        sl = slice(int(cu[p]), int(cu[p + 1]))
        t = int(pl["task"][p])
        y, k, v = O.layer(spec, W_np, oracle_adapter(model.adapters[0], t), x_in[sl], pos=pl["pos"][sl])
        i = int(pl["order"][p])
        s0, n = int(kvs[i]), int(lens[i])
        worst = max(worst, O.row_rel_error(got[sl], y), O.row_rel_error(k_all[s0:s0 + n], k),
                    O.row_rel_error(v_all[s0:s0 + n], v))
        written[s0:s0 + n] = True
    log(f"  max row rel err (output, cached k, cached v) {worst:.3e}")
    assert worst < tol(w)
    assert np.all(k_all[~written] == sentinel) and np.all(v_all[~written] == sentinel)


def test_attach_and_remove_adapter_between_batches():
    """Task extensions are replaced at run time without touching the
    backbone: vfm_lora_attach gives task 5 a new rank-8 adapter, then removes
    it.  After each change the task's rows match the oracle with its new
    adapter (or the bare backbone), and every other task's rows stay
    bit-identical to the first run.  ViT-B layer, tasks 5, 0, 5, 2, 9, 0."""
    w, batch, model, inp, kv, pb, fwd, pl = _setup(2, n_layers=1, b_std=0.1)
    x_in = as_f32(expected_embed(w, batch, inp, pl))
    set_rows(fwd.x, x_in)
    x0 = fwd.x.clone()
    spec = spec_of(w)
    W_np = oracle_weights(model.layers[0])
    cu = pl["cu_seqlens"]
    tasks = [int(pl["task"][p]) for p in range(batch.n_req)]

    def run():
        fwd.x.copy_(x0)
        fwd.layer(0)
        torch.cuda.synchronize()
        return fwd.x.double().cpu().numpy()

    first = run()
    g = torch.Generator(device="cuda").manual_seed(11)
    r, sc = 8, 1.5
    A = {p: (torch.randn(r, w.d, generator=g, device="cuda") / w.d ** 0.5).to(torch.bfloat16)
         for p in ("q", "k", "v", "o")}
    Bm = {p: (0.1 * torch.randn(w.d, r, generator=g, device="cuda")).to(torch.bfloat16)
          for p in ("q", "k", "v", "o")}
    new_ad = {p: (np64(A[p]), np64(Bm[p]), sc) for p in A}
    for stage, ad5 in (("attach", new_ad), ("remove", None)):
        if ad5 is None:
            B.vfm_lora_attach(model.lora[0], 5, 0, 0.0)
        else:
            B.vfm_lora_attach(model.lora[0], 5, r, sc, A, Bm)
        got = run()
        worst = 0.0
        for p in range(batch.n_req):
            sl = slice(int(cu[p]), int(cu[p + 1]))
            if tasks[p] == 5:
                y = O.layer(spec, W_np, ad5, x_in[sl], pos=pl["pos"][sl])[0]
                worst = max(worst, O.row_rel_error(got[sl], y))
            else:
                assert np.array_equal(got[sl], first[sl]), (stage, p)
        log(f"  {stage}: task 5 max row rel err {worst:.3e}")
        assert worst < tol(w)
    # cost of one table update (host call + its one-thread kernel)
    import time
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(200):
        B.vfm_lora_attach(model.lora[0], 5, r if i % 2 else 0, sc, A, Bm)
    torch.cuda.synchronize()
    log(f"  attach / remove: {(time.perf_counter() - t0) / 200 * 1e6:.1f} us per call")


def test_attach_head_between_batches():
    """vfm_head_attach swaps task 2's head for a new 17-output one: the next
    batch (planned with the new width) gives the oracle's logits for task 2
    and the unchanged ones for the other tasks."""
    w, batch, model, inp, kv, pb, fwd, pl = _setup(2, n_layers=1)
    x_fin = seeded_rows(pb.T, w.d, 202)            # the final hidden rows, plan order
    set_rows(fwd.x, x_fin)
    fwd.head()
    torch.cuda.synchronize()
    out_a = fwd.out.cpu().numpy()
    n_out = model.heads.n_out.copy()
    g = torch.Generator(device="cuda").manual_seed(5)
    Wn = (torch.randn(17, w.d, generator=g, device="cuda") / w.d ** 0.5).to(torch.bfloat16)
    bn = (0.02 * torch.randn(17, generator=g, device="cuda")).to(torch.bfloat16)
    B.vfm_head_attach(model.head_tab, 2, 17, Wn, bn)
    n_out[2] = 17
    pb2 = B.Batch(batch.task_id, batch.seq_len, w.n_tasks, n_out=n_out)
    fwd2 = R.Forward(model, pb2, inp)
    fwd2.x.copy_(fwd.x)
    fwd2.head()
    torch.cuda.synchronize()
    out_b = fwd2.out.cpu().numpy()
    heads_np = [(np64(model.heads.W[t]), np64(model.heads.b[t])) for t in range(w.n_tasks)]
    heads_np[2] = (np64(Wn), np64(bn))
    pl2 = oracle_plan(w, batch, n_out)
    off_a, off_b = pl["logit_off"], pl2["logit_off"]
    for i in range(batch.n_req):
        t = int(batch.task_id[i])
        ob = out_b[off_b[i]:off_b[i + 1]]
        if t == 2:
            p = int(np.nonzero(pl2["order"] == i)[0][0])
            sl = slice(int(pl2["cu_seqlens"][p]), int(pl2["cu_seqlens"][p + 1]))
            xn = O.final(spec_of(w), np64(model.final["w"]), np64(model.final["b"]), x_fin[sl])
            ref = O.head(O.pool(xn, w.pool), heads_np[2][0], heads_np[2][1])
            assert len(ob) == 17 and O.row_rel_error(ob[None], ref[None]) < tol(w)
        else:
            assert np.array_equal(ob, out_a[off_a[i]:off_a[i + 1]])


@pytest.mark.parametrize("idx,act", [(3, B.VFM_ACT_GELU), (1, B.VFM_ACT_RELU)])
def test_mlp_decoder_heads(idx, act):
    """Per-task two-layer MLP decoder heads (hidden width 128) mixed with
    linear ones in one batch: every request's outputs against the oracle's
    act(pooled W1^T + b1) W^T + b (or W pooled + b for the linear tasks)."""
    w, batch, model, inp, kv, pb, fwd, pl = _setup(idx, n_layers=1)
    hd = model.heads
    dt = w.torch_dtype
    g = torch.Generator(device="cuda").manual_seed(21)
    H = 128
    W1s, b1s, Ws, bs = [], [], [], []
    for t in range(w.n_tasks):
        n = int(hd.n_out[t])
        if t % 2:      # MLP head
            W1s.append((torch.randn(H, w.d, generator=g, device="cuda") / w.d ** 0.5).to(dt))
            b1s.append((0.1 * torch.randn(H, generator=g, device="cuda")).to(dt))
            Ws.append((torch.randn(n, H, generator=g, device="cuda") / H ** 0.5).to(dt))
        else:          # linear head, as drawn by the workload
            W1s.append(None)
            b1s.append(None)
            Ws.append(hd.W[t])
        bs.append(hd.b[t])
    tab = B.HeadTable(hd.n_out, Ws, bs, model.head_tab.c.pool, W1s=W1s, b1s=b1s, hidden=H, act=act)
    model.head_tab = tab
    x_fin = seeded_rows(pb.T, w.d, 300 + idx)      # the final hidden rows, plan order
    set_rows(fwd.x, x_fin)
    fwd.head()
    torch.cuda.synchronize()
    out = fwd.out.cpu().numpy()
    spec = spec_of(w)
    fw = np64(model.final["w"])
    fb = np64(model.final["b"]) if model.final.get("b") is not None else None
    cu, off = pl["cu_seqlens"], pl["logit_off"]
    worst = 0.0
    for p in range(batch.n_req):
        i, t = int(pl["order"][p]), int(pl["task"][p])
        pooled = O.pool(O.final(spec, fw, fb, x_fin[int(cu[p]):int(cu[p + 1])]), w.pool)
        if t % 2:
            ref = O.head_mlp(pooled, np64(W1s[t]), np64(b1s[t]), np64(Ws[t]), np64(bs[t]),
                             act="gelu" if act == B.VFM_ACT_GELU else "relu")
        else:
            ref = O.head(pooled, np64(Ws[t]), np64(bs[t]))
        worst = max(worst, O.row_rel_error(out[off[i]:off[i + 1]][None], ref[None]))
    log(f"  MLP / linear heads, workload {idx}: max rel err {worst:.3e}")
    assert worst < tol(w)
    # attach an MLP head to task 0 (linear so far) between batches: task 0's
    # outputs follow the new head, every other task's stay bit-identical
    n0 = int(hd.n_out[0])
    W1n = (torch.randn(H, w.d, generator=g, device="cuda") / w.d ** 0.5).to(dt)
    b1n = (0.1 * torch.randn(H, generator=g, device="cuda")).to(dt)
    Wn = (torch.randn(n0, H, generator=g, device="cuda") / H ** 0.5).to(dt)
    B.vfm_head_attach(tab, 0, n0, Wn, hd.b[0], W1n, b1n)
    fwd.head()
    torch.cuda.synchronize()
    out2 = fwd.out.cpu().numpy()
    for p in range(batch.n_req):
        i, t = int(pl["order"][p]), int(pl["task"][p])
        sl = slice(off[i], off[i + 1])
        if t == 0:
            pooled = O.pool(O.final(spec, fw, fb, x_fin[int(cu[p]):int(cu[p + 1])]), w.pool)
            ref = O.head_mlp(pooled, np64(W1n), np64(b1n), np64(Wn), np64(hd.b[0]),
                             act="gelu" if act == B.VFM_ACT_GELU else "relu")
            assert O.row_rel_error(out2[sl][None], ref[None]) < tol(w)
        else:
            assert np.array_equal(out2[sl], out[sl])


def _expected_series_rows(batch, pl, src, C_, patch, Ws, bs, W_pe, b_pe):
    """Oracle rows (plan order): each request's channels combined by its
    task's encoder (or channel 0 without one), patched and embedded."""
    cu_o = pl["cu_orig"]
    rows = []
    for p, i in enumerate(pl["order"]):
        t = int(pl["task"][p])
        L = int(batch.seq_len[i]) * patch
        xr = src[C_ * int(cu_o[i]) * patch:C_ * int(cu_o[i + 1]) * patch].reshape(C_, L)
        s = O.channel_combine(xr, Ws[t], bs[t]) if Ws[t] is not None else xr[0]
        rows.append(O.patch_embed(s, patch, W_pe, b_pe))
    return np.concatenate(rows)


@pytest.mark.parametrize("idx", [3, 1])
def test_channel_encoder_embed(idx):
    """Per-task linear channel combiners (3 channels to 1) fused with the
    shared patch embedding, tasks with an even id carrying one and the others
    feeding channel 0: every row against the oracle's combine -> patch ->
    embed; then an encoder attached to task 1 and removed from task 0 between
    batches, the other tasks' rows bit-identical."""
    w, batch, model, inp, kv, pb, fwd, pl = _setup(idx)
    C_, patch = 3, 8
    src, W_pe, b_pe = wl.multichannel_series_inputs(w, batch, C_, patch, "cuda")
    g = torch.Generator(device="cuda").manual_seed(31)
    Ws = [torch.randn(C_, generator=g, device="cuda") if t % 2 == 0 else None for t in range(w.n_tasks)]
    bs = [0.1 * torch.randn(1, generator=g, device="cuda") if t % 2 == 0 else None for t in range(w.n_tasks)]
    enc = B.EncoderTable(C_, Ws, bs)
    log(f"series encoder workload {idx} T={pb.T} channels {C_}")
    x = torch.empty(pb.T, w.d, dtype=torch.float32, device="cuda")
    B.vfm_embed_series(model.cfg, pb.c, enc, src, patch, W_pe, b_pe, x)
    torch.cuda.synchronize()
    src_np, Wpe_np, bpe_np = np64(src), np64(W_pe), np64(b_pe)
    Ws_np, bs_np = [np64(v) for v in Ws], [np64(v) for v in bs]
    got = x.double().cpu().numpy()
    ref = _expected_series_rows(batch, pl, src_np, C_, patch, Ws_np, bs_np, Wpe_np, bpe_np)
    err = O.row_rel_error(got, ref)
    log(f"  max rel err {err:.3e}")
    assert err < 1e-5
    # encoder lifecycle between batches
    Wn = torch.tensor([0.5, -1.0, 2.0], device="cuda")
    bn = torch.tensor([0.25], device="cuda")
    B.vfm_encoder_attach(enc, 1, Wn, bn)
    B.vfm_encoder_attach(enc, 0, None)
    x2 = torch.empty_like(x)
    B.vfm_embed_series(model.cfg, pb.c, enc, src, patch, W_pe, b_pe, x2)
    torch.cuda.synchronize()
    Ws_np[1], bs_np[1] = np64(Wn), np64(bn)
    Ws_np[0], bs_np[0] = None, None
    got2 = x2.double().cpu().numpy()
    ref2 = _expected_series_rows(batch, pl, src_np, C_, patch, Ws_np, bs_np, Wpe_np, bpe_np)
    assert O.row_rel_error(got2, ref2) < 1e-5
    other = pl["task"][pl["row_req"]] >= 2
    assert np.array_equal(got2[other], got[other])


@pytest.mark.parametrize("page", [16, 64])
def test_paged_decode_matches_contiguous(page):
    """A decode layer over a paged cache (pages in random order, spare pages
    in the pool) gives bit-identical rows to the same layer over the
    contiguous head-major cache, and writes the new token's K / V into its
    page.  Contexts 0, 63, 300, 64 and 4200 (three 2048-key chunks)."""
    w, batch, model, inp, kv, pb, fwd, pl = _setup(5)
    log(f"paged decode, page {page}, ctx {list(batch.ctx)}")
    fwd.embed()
    x0 = fwd.x.clone()
    n_tok = batch.ctx.astype(np.int64) + 1
    kp, vp, table = R.paged_from_contiguous(kv.k[0], kv.v[0], kv.kv_start, n_tok, page,
                                            np.random.default_rng(page), spare_pages=7)
    pkv = B.PagedKV(kp, vp, page, table)
    fwd.layer(0)
    torch.cuda.synchronize()
    x_c = fwd.x.clone()
    fwd.x.copy_(x0)
    B.vfm_layer_forward_paged(model.cfg, model.c_layers[0], model.lora_c(0), pb.c, fwd.x, pkv, fwd.ws)
    torch.cuda.synchronize()
    assert torch.equal(fwd.x, x_c)
    for i in range(batch.n_req):
        c = int(batch.ctx[i])
        ps = int(table[i, c // page]) * page + c % page
        cs = int(kv.kv_start[i]) + c
        assert torch.equal(kp[:, ps], kv.k[0][:, cs]) and torch.equal(vp[:, ps], kv.v[0][:, cs])


def _page_rows(pool, table, i, n, page):
    """Positions 0 .. n-1 of request i from a paged pool, as [n, n_heads * head_dim]."""
    pos = np.arange(n)
    phys = table[i, pos // page].astype(np.int64) * page + pos % page
    rows = pool[:, torch.from_numpy(phys).to(pool.device)]
    return rows.permute(1, 0, 2).reshape(n, -1)


@pytest.mark.parametrize("ctx_long,layout", [(300, "paged"), (2100, "paged"), (2100, "contiguous"),
                                             (0, "causal-paged"), (300, "paged-chunked"),
                                             (2100, "contiguous-chunked")])
def test_mixed_step_over_cache(ctx_long, layout):
    """One continuous-batching step (7B decoder layer dims): two prompts (70
    and 33 tokens, ctx 0) and three decode tokens (ctx 63, 1100 and a long
    one) in one batch, over a paged cache (pages of 64 in random order) or
    the contiguous one (vfm_layer_forward, slots kv_start + k), with and
    without a 40-row prompt chunk after cached tokens in place of a decode
    row; and a prompts-only causal step over pages.  Every row against the oracle
    (prompts causal over themselves, decode rows over their cached keys plus
    themselves), and every new row's rotated K and V in its slots."""
    w = wl.WORKLOADS[4]
    task_id = np.array([3, 0, 3, 63, 5], np.int32)
    if layout == "causal-paged":
        seq_len = np.array([70, 1, 33, 5, 2], np.int32)
        ctx = np.zeros(5, np.int32)
    else:
        # "-chunked": request 3 is a 40-row prompt chunk after its ctx cached tokens
        seq_len = np.array([70, 1, 33, 40 if "chunked" in layout else 1, 1], np.int32)
        ctx = np.array([0, 63, 0, ctx_long, 1100], np.int32)
    worst = _run_mixed_step(w, task_id, seq_len, ctx, layout)
    assert worst < tol(w)


# A 1024-wide decoder with 16 heads of 64 dims (the head_dim-64 kernels);
# the 7B one has 32 heads of 128.
DECODER_DH64 = dict(d=1024, n_heads=16, head_dim=64, d_ff=2816)


@pytest.mark.parametrize("dh,layout", [(128, "paged"), (128, "contiguous"), (64, "paged"), (64, "contiguous")])
def test_long_prompt_chunks_over_cache(dh, layout):
    """Chunked prefill in the cache-reading flash kernel away from its easy
    case: a 170-row prompt chunk after 333 cached tokens (three 64-query
    blocks, so q0 > 0, and a context that is not a multiple of 64) and a
    65-row chunk after 100, next to a 300-row prompt (so the first pass is
    the flash kernel, not the short one) and a decode row at ctx 1100; head
    dims 128 and 64, pages of 64 in random order or the contiguous cache.
    Every row against the oracle with those cached keys, and every new K /
    V row in its slots."""
    w = wl.WORKLOADS[4]
    if dh == 64:
        w = w.replace(**DECODER_DH64)
    task_id = np.array([3, 0, 63, 3, 5], np.int32)
    seq_len = np.array([300, 170, 1, 65, 2], np.int32)
    ctx = np.array([0, 333, 1100, 100, 0], np.int32)
    worst = _run_mixed_step(w, task_id, seq_len, ctx, layout)
    assert worst < tol(w)


def _run_mixed_step(w, task_id, seq_len, ctx, layout):
    """One mixed (or, for "causal-paged", prompts-only causal) step of one
    decoder layer over a paged or contiguous cache holding seeded K / V;
    checks every new K / V row and returns the worst row error of the
    layer's output against the oracle."""
    batch = wl.Batch(task_id, seq_len, ctx)
    model = R.Model(w, n_layers=1, b_std=0.1)
    inp = R.Inputs(w, batch)
    n_tok = ctx.astype(np.int64) + seq_len
    if layout.startswith("contiguous"):
        # slots kv_start[i] + k: a "page table" of single slots for the oracle's reads
        page = 1
        kvs = np.concatenate([[0], np.cumsum(n_tok + 3)[:-1]]).astype(np.int32)
        total = int((n_tok + 3).sum())
        table = kvs[:, None] + np.arange(int(n_tok.max()), dtype=np.int32)[None, :]
    else:
        page = 64
        need = (n_tok + page - 1) // page
        total = int(need.sum()) + 5
        perm = np.random.default_rng(11).permutation(total).astype(np.int32)
        table = np.zeros((len(n_tok), int(need.max())), np.int32)
        first = np.concatenate([[0], np.cumsum(need)[:-1]])
        for i in range(len(n_tok)):
            table[i, :need[i]] = perm[first[i]:first[i] + need[i]]
    g = torch.Generator(device="cuda").manual_seed(13)
    kp = torch.randn(w.n_heads, total * page, w.head_dim, generator=g, device="cuda").to(torch.bfloat16)
    vp = torch.randn(w.n_heads, total * page, w.head_dim, generator=g, device="cuda").to(torch.bfloat16)
    cfg = R.cfg_for(w)
    cfg.attn = B.VFM_ATTN_CAUSAL if layout == "causal-paged" else B.VFM_ATTN_MIXED
    contiguous = layout.startswith("contiguous")
    pb = B.Batch(task_id, seq_len, w.n_tasks, ctx_len=ctx, kv_start=kvs if contiguous else None)
    fwd = R.Forward(model, pb, inp)
    ws = torch.empty(B.vfm_workspace_size(cfg, pb.c, model.lora_c(0)), dtype=torch.uint8, device="cuda")
    log(f"{layout} step: lens {list(seq_len)} ctx {list(ctx)} T={pb.T}")
    pl = O.plan(task_id, seq_len, w.n_tasks, ctx=ctx)
    x_in = as_f32(expected_embed(w, batch, inp, pl))
    set_rows(fwd.x, x_in)
    if contiguous:
        B.vfm_layer_forward(cfg, model.c_layers[0], model.lora_c(0), pb.c, fwd.x, kp, vp, total, ws)
    else:
        B.vfm_layer_forward_paged(cfg, model.c_layers[0], model.lora_c(0), pb.c, fwd.x,
                                  B.PagedKV(kp, vp, page, table), ws)
    torch.cuda.synchronize()
    got = fwd.x.double().cpu().numpy()
    spec = spec_of(w)
    W_np = oracle_weights(model.layers[0])
    cu = pl["cu_seqlens"]
    worst = 0.0
    for p in range(batch.n_req):
        sl = slice(int(cu[p]), int(cu[p + 1]))
        i, t = int(pl["order"][p]), int(pl["task"][p])
        c, L = int(ctx[i]), int(seq_len[i])
        kvp = None
        if c > 0:
            kvp = (np64(_page_rows(kp, table, i, c, page)), np64(_page_rows(vp, table, i, c, page)))
        y, k, v = O.layer(spec, W_np, oracle_adapter(model.adapters[0], t), x_in[sl], pos=pl["pos"][sl], kv=kvp)
        worst = max(worst, O.row_rel_error(got[sl], y))
        k_new = np64(_page_rows(kp, table, i, c + L, page))[c:]
        v_new = np64(_page_rows(vp, table, i, c + L, page))[c:]
        assert O.row_rel_error(k_new, k) < tol(w) and O.row_rel_error(v_new, v) < tol(w)
    log(f"  max rel err {worst:.3e}")
    return worst


@pytest.mark.parametrize("idx,seed", [(1, 0), (1, 1), (1, 2), (2, 3), (2, 4), (3, 5), (2, 6)])
def test_random_batches_layer_parity(idx, seed):
    """Seeded random batches: 1..12 requests of 1..150 rows, task ids drawn
    over every task (absent ids included), per-task ranks 0 / 8 / 16: every
    row of one layer against the oracle, both sides fed the oracle's input
    rows (small batches take the split-K path, larger ones the tile path)."""
    w = wl.WORKLOADS[idx]
    rng = np.random.default_rng(1000 + seed)
    big = seed == 6                            # at least 1024 rows: the large-tile path
    n = 12 if big else int(rng.integers(1, 13))
    case = dict(task_id=rng.integers(0, w.n_tasks, size=n).tolist(),
                seq_len=rng.integers(90 if big else 1, 151, size=n).tolist())
    ranks = (8 * rng.integers(0, 3, size=w.n_tasks)).astype(np.int32)
    if idx == 3:
        case["seq_len"] = [64] * n             # the time-series workload's patches come in whole series
    w_, batch, model, inp, kv, pb, fwd, pl = _setup(idx, n_layers=1, b_std=0.1, ranks=ranks, case=case)
    log(f"random batch workload {idx} seed {seed}: {n} requests, T={pb.T}, ranks {list(ranks[:8])}")
    assert not big or pb.T >= B.VFM_SMALL_BATCH_ROWS
    x_in = as_f32(expected_embed(w, batch, inp, pl))
    set_rows(fwd.x, x_in)
    fwd.layer(0)
    torch.cuda.synchronize()
    got = fwd.x.double().cpu().numpy()
    res = oracle_layer_rows(w, oracle_weights(model.layers[0]), model.adapters[0], pl, x_in, range(batch.n_req))
    cu = pl["cu_seqlens"]
    worst = max(O.row_rel_error(got[cu[p]:cu[p + 1]], res[p][0]) for p in range(batch.n_req))
    log(f"  max row rel err {worst:.3e}")
    assert worst < tol(w)
