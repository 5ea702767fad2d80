"""GPU tests of continuous batching over a paged KV cache: a small decoder
FM (two layers, d 256, per-task LoRA on every projection and a per-task LM
head over a 256-token vocabulary) serves requests of ragged prompt lengths
and output budgets that join and leave the running batch at different
steps.  The oracle decodes every request greedily on its own (fp64, from the
prompt); each step's head outputs of each request are checked against the
oracle's for as long as the two runs have picked the same tokens, and a
different pick must be a near-tie of the oracle's outputs."""
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


def _oracle_greedy(w, model, emb_np, task, prompt, n_new):
    """The oracle's own greedy decode of one request: n_new steps, each a
    causal forward over the prompt and the oracle's earlier picks (the
    request's task adapters and head), returning the picks and each step's
    head outputs at the last position."""
    spec = spec_of(w)
    layers = [oracle_weights(model.layers[li]) for li in range(model.n_layers)]
    ads = [oracle_adapter(model.adapters[li], task) for li in range(model.n_layers)]
    fw, fb = np64(model.final["w"]), np64(model.final.get("b"))
    W, b = np64(model.heads.W[task]), np64(model.heads.b[task])
    tokens, picks, outs = list(prompt), [], []
    for _ in range(n_new):
        x = emb_np[np.asarray(tokens)]
        pos = np.arange(len(tokens))
        for li in range(model.n_layers):
            x, _, _ = O.layer(spec, layers[li], ads[li], x, pos=pos)
        logits = O.head(O.final(spec, fw, fb, x)[-1], W, b)
        outs.append(logits)
        picks.append(int(np.argmax(logits)))
        tokens.append(picks[-1])
    return picks, outs


@pytest.mark.parametrize("dtype,page,sched", [("bf16", 16, "fifo"), ("f32", 32, "fifo"), ("bf16", 16, "bfq"),
                                             ("bf16", 16, "fifo-chunked")])
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
    # "-chunked": 20 tokens per step, so the 24- and 33-token prompts are fed in chunks
    budget = 20 if sched.endswith("chunked") else 96
    cb = R.ContinuousBatcher(model, emb, page_size=page, n_pages=12, max_seqs=3, max_step_tokens=budget,
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
    worst, compared = 0.0, 0
    for rid, (task, L, n_new) in enumerate(REQUESTS):
        gen = done[rid]
        assert len(gen) == n_new and len(outs[rid]) == n_new
        ref_picks, ref = _oracle_greedy(w, model, emb_np, task, prompts[rid], n_new)
        # step j of both runs has the same input tokens while the picks agree
        for j in range(n_new):
            got = outs[rid][j]
            worst = max(worst, O.row_rel_error(got[None], ref[j][None]))
            compared += 1
            # the greedy kernel's pick is the first maximum of the step's outputs
            assert gen[j] == int(np.argmax(got))
            if gen[j] != ref_picks[j]:
                # a different pick is only allowed at a near-tie of the oracle's outputs;
                # past it the two runs decode different tokens
                assert ref[j][gen[j]] >= ref[j].max() - tol(w) * np.abs(ref[j]).max()
                break
    log(f"  {compared} of {sum(n for _, _, n in REQUESTS)} steps compared, max rel err {worst:.3e}")
    assert worst < tol(w)
    if w.dtype == "f32":
        assert compared == sum(n for _, _, n in REQUESTS)
    # the same requests through the asynchronous path (no per-step read-back)
    # pick the same tokens
    bfq2 = B.BFQ([1.0, 2.0, 1.0], np.linspace(1.0, 2.0, 3), b_max=2) if sched == "bfq" else None
    cb2 = R.ContinuousBatcher(model, emb, page_size=page, n_pages=12, max_seqs=3, max_step_tokens=budget,
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
