"""GPU tests of continuous batching over a paged KV cache: a small decoder
FM (two layers, d 256, per-task LoRA on every projection and a per-task LM
head over a 256-token vocabulary) serves requests of ragged prompt lengths
and output budgets that join and leave the running batch at different
steps.  Every step's head outputs of every request are checked against the
oracle's causal forward over the same tokens, and every greedy pick against
the step's own outputs."""
import numpy as np
import pytest
import torch

from oracle import vfm_oracle as O
from paper_2606_09643_amd import binding as B
from paper_2606_09643_amd import runner as R
from paper_2606_09643_amd import workloads as wl
from tests.gpu_common import log, tol
from tests.helpers import np64, oracle_adapter, oracle_weights, spec_of

pytestmark = pytest.mark.gpu


def _tiny_decoder(dtype):
    return wl.Workload(6, f"tiny-decoder-{dtype}", dtype, "decoder", 2, 256, 2, 128, 512,
                       n_tasks=3, n_req=6, rank=8, lora_targets=wl.PROJ, lora_scale=2.0, zipf_s=None,
                       seq_len=(1, 40), mode="prefill", ctx=None, inputs="tokens", pool="last",
                       head="fixed:256", vocab=256)


REQUESTS = [  # (task, prompt length, new tokens)
    (0, 5, 6), (2, 17, 3), (1, 1, 8), (0, 33, 4), (2, 9, 5), (1, 24, 7)]


def _oracle_logits(w, model, emb_np, task, tokens, n_prompt):
    """Head outputs at positions n_prompt - 1 .. len(tokens) - 1 of the
    oracle's causal forward over `tokens` (the request's task adapters and
    head)."""
    spec = spec_of(w)
    x = emb_np[np.asarray(tokens)]
    pos = np.arange(len(tokens))
    for li in range(model.n_layers):
        x, _, _ = O.layer(spec, oracle_weights(model.layers[li]), oracle_adapter(model.adapters[li], task), x,
                          pos=pos)
    xn = O.final(spec, np64(model.final["w"]), np64(model.final.get("b")), x)
    W, b = np64(model.heads.W[task]), np64(model.heads.b[task])
    return [O.head(xn[j], W, b) for j in range(n_prompt - 1, len(tokens))]


@pytest.mark.parametrize("dtype,page,sched", [("bf16", 16, "fifo"), ("f32", 32, "fifo"), ("bf16", 16, "bfq")])
def test_continuous_batching_loop(dtype, page, sched):
    w = _tiny_decoder(dtype)
    model = R.Model(w, n_layers=2, b_std=0.1)
    one = wl.Batch(np.zeros(1, np.int32), np.ones(1, np.int32), None)
    _, emb = wl.token_inputs(w, one, "cuda")
    rng = np.random.default_rng(5)
    prompts = [rng.integers(0, w.vocab, size=L).astype(np.int32) for _, L, _ in REQUESTS]
    bfq = None
    if sched == "bfq":
        bfq = B.BFQ([1.0, 2.0, 1.0], np.linspace(1.0, 2.0, 3), b_max=2)
    # three sequence slots and a 12-page pool: requests wait for slots and pages
    cb = R.ContinuousBatcher(model, emb, page_size=page, n_pages=12, max_seqs=3, max_step_tokens=96,
                             max_pages=6, bfq=bfq, record=True)
    for rid, ((task, _, n_new), pr) in enumerate(zip(REQUESTS, prompts)):
        cb.submit(rid, task, pr, n_new)
    log(f"loop {dtype} page {page} {sched}")
    done = cb.run()
    log(f"  {cb.steps} steps")
    assert sorted(done) == list(range(len(REQUESTS)))
    assert cb.alloc.count(0)[1] == 12                     # every page back in the pool
    # per request, its head outputs step by step
    outs = {rid: [] for rid in done}
    for step in cb.trace:
        for rid, o in step:
            outs[rid].append(o)
    emb_np = np64(emb)
    worst = 0.0
    for rid, (task, L, n_new) in enumerate(REQUESTS):
        gen = done[rid]
        assert len(gen) == n_new and len(outs[rid]) == n_new
        tokens = np.concatenate([prompts[rid], np.asarray(gen[:-1], np.int32)])
        ref = _oracle_logits(w, model, emb_np, task, tokens, L)
        for j in range(n_new):
            got = outs[rid][j]
            worst = max(worst, O.row_rel_error(got[None], ref[j][None]))
            # the greedy pick is the first maximum of the step's own outputs
            assert gen[j] == int(np.argmax(got))
            # and a maximum of the oracle's outputs up to the tolerance
            assert ref[j][gen[j]] >= ref[j].max() - tol(w) * np.abs(ref[j]).max()
    log(f"  max rel err {worst:.3e}")
    assert worst < tol(w)
    # the same requests through the asynchronous path (no per-step read-back)
    # pick the same tokens
    bfq2 = B.BFQ([1.0, 2.0, 1.0], np.linspace(1.0, 2.0, 3), b_max=2) if sched == "bfq" else None
    cb2 = R.ContinuousBatcher(model, emb, page_size=page, n_pages=12, max_seqs=3, max_step_tokens=96,
                              max_pages=6, bfq=bfq2)
    for rid, ((task, _, n_new), pr) in enumerate(zip(REQUESTS, prompts)):
        cb2.submit(rid, task, pr, n_new)
    assert cb2.run() == done and cb2.steps == cb.steps


def test_greedy_tokens_ties_nan_and_empty():
    """vfm_greedy_tokens: first maximum on ties, NaN never chosen, -inf
    allowed, a request without outputs gets -1; against numpy's argmax of
    the same fp32 values."""
    n_out = np.array([5, 0, 300, 1, 64], np.int32)
    pb = B.Batch(np.arange(5, dtype=np.int32), np.ones(5, np.int32), 5, n_out=n_out)
    off = pb.out_off()
    rng = np.random.default_rng(3)
    out = rng.normal(size=int(off[-1])).astype(np.float32)
    out[off[0]:off[1]] = [1.0, 3.0, np.nan, 3.0, 2.0]            # tie: index 1
    out[off[2] + 17] = np.inf
    out[off[2] + 200] = np.inf                                  # tie at +inf: 17
    out[off[3]] = -np.inf                                       # the only output
    out[off[4]:off[5]] = np.nan
    out[off[4] + 40] = 0.5                                      # the only number
    ids = torch.full((5,), 99, dtype=torch.int32, device="cuda")
    B.vfm_greedy_tokens(pb.c, torch.from_numpy(out).cuda(), ids)
    assert ids.cpu().tolist() == [1, -1, 17, 0, 40]
    big = rng.normal(size=(64, 4096)).astype(np.float32)
    pb2 = B.Batch(np.zeros(64, np.int32), np.ones(64, np.int32), 1, n_out=np.array([4096], np.int32))
    ids2 = torch.empty(64, dtype=torch.int32, device="cuda")
    B.vfm_greedy_tokens(pb2.c, torch.from_numpy(big.ravel()).cuda(), ids2)
    assert np.array_equal(ids2.cpu().numpy(), big.argmax(axis=1))
