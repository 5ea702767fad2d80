"""Pins of the fp64 oracle against things other than itself (CPU only).

Each pin is chosen so that a plausible slip in the oracle (a dropped term, a
wrong sign or index, a transposed operand) fails at least one of them:
library routines (torch's TransformerEncoderLayer, transformers'
LlamaDecoderLayer and rotary helpers, F.scaled_dot_product_attention,
F.layer_norm / F.rms_norm / F.gelu / F.silu), brute force, closed forms and
the invariants the paper's deployment sharing must keep (Section 2.3;
Section 4.2 adapter handling).
"""
import itertools
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import vfm_oracle as O
from paper_2606_09643_amd import workloads as wl
from tests.helpers import np64, oracle_adapter, oracle_weights, spec_of

pytestmark = pytest.mark.filterwarnings("ignore::UserWarning")


def _rng(seed=0):
    return np.random.default_rng(seed)


# --------------------------------------------------------------------------
# plan: brute force with a library stable sort
# --------------------------------------------------------------------------
def _brute_plan(task_id, seq_len, n_tasks, ctx=None, n_out=None):
    task_id = np.asarray(task_id)
    seq_len = np.asarray(seq_len)
    order = np.argsort(task_id, kind="stable")
    cu = np.concatenate([[0], np.cumsum(seq_len[order])])
    seg_req = np.searchsorted(task_id[order], np.arange(n_tasks + 1), side="left")
    seg_req[-1] = len(task_id)
    seg_row = cu[seg_req]
    pos = np.concatenate([np.arange(seq_len[i]) + (ctx[i] if ctx is not None else 0)
                          for i in order]) if len(order) else np.zeros(0)
    row_req = np.repeat(np.arange(len(order)), seq_len[order])
    widths = np.asarray(n_out)[task_id] if n_out is not None else np.zeros(len(task_id))
    return {"order": order, "cu_seqlens": cu, "seg_req": seg_req, "seg_row": seg_row,
            "pos": pos, "row_req": row_req,
            "cu_orig": np.concatenate([[0], np.cumsum(seq_len)]),
            "logit_off": np.concatenate([[0], np.cumsum(widths)]),
            "task": task_id[order]}


def _check_plan(task_id, seq_len, n_tasks, ctx=None, n_out=None):
    got = O.plan(task_id, seq_len, n_tasks, ctx=ctx, n_out=n_out)
    ref = _brute_plan(task_id, seq_len, n_tasks, ctx=ctx, n_out=n_out)
    for k, v in ref.items():
        assert np.array_equal(got[k], np.asarray(v, np.int64)), k


def test_plan_exhaustive_small():
    r = _rng(1)
    for n_tasks in (1, 2, 3):
        for n_req in range(1, 6):
            for tid in itertools.product(range(n_tasks), repeat=n_req):
                lens = r.integers(1, 5, size=n_req)
                _check_plan(tid, lens, n_tasks, n_out=r.integers(1, 4, size=n_tasks))


def test_plan_edge_cases():
    r = _rng(2)
    _check_plan([0] * 7, [3] * 7, 1)                      # one task
    _check_plan([5] * 4, [1, 2, 3, 4], 8)                 # all tasks but one empty
    _check_plan([2], [9], 3)                              # one request
    tid = r.integers(0, 128, size=256)
    ctx = r.integers(256, 2049, size=256)
    _check_plan(tid, np.ones(256, int), 128, ctx=ctx, n_out=np.full(128, 8))
    with pytest.raises(ValueError):
        O.plan([0, 3], [1, 1], 3)


# --------------------------------------------------------------------------
# elementary ops vs library routines and special cases
# --------------------------------------------------------------------------
def test_norms_vs_torch():
    r = _rng(3)
    x = r.normal(size=(7, 48))
    g = 1 + 0.1 * r.normal(size=48)
    b = 0.1 * r.normal(size=48)
    ref = F.layer_norm(torch.from_numpy(x), (48,), torch.from_numpy(g), torch.from_numpy(b), 1e-5)
    assert np.allclose(O.layer_norm(x, g, b, 1e-5), ref.numpy(), rtol=0, atol=1e-12)
    ref = F.rms_norm(torch.from_numpy(x), (48,), torch.from_numpy(g), 1e-6)
    assert np.allclose(O.rms_norm(x, g, 1e-6), ref.numpy(), rtol=0, atol=1e-12)
    # LayerNorm of a constant row is exactly its shift
    c = np.full((1, 48), 3.25)
    assert np.allclose(O.layer_norm(c, g, b, 1e-5), b[None, :], atol=1e-12)


def test_activations_vs_torch():
    x = np.linspace(-8, 8, 1001)
    t = torch.from_numpy(x)
    assert np.allclose(O.gelu(x), F.gelu(t).numpy(), atol=1e-14)
    assert np.allclose(O.silu(x), F.silu(t).numpy(), atol=1e-14)


@pytest.mark.parametrize("causal", [False, True])
def test_attention_vs_sdpa(causal):
    r = _rng(4)
    H, dh, L = 3, 16, 11
    q, k, v = (r.normal(size=(L, H * dh)) for _ in range(3))
    got = O.attention(q, k, v, H, dh, causal=causal)
    tq, tk, tv = (torch.from_numpy(a).view(L, H, dh).transpose(0, 1) for a in (q, k, v))
    ref = F.scaled_dot_product_attention(tq, tk, tv, is_causal=causal)
    assert np.allclose(got, ref.transpose(0, 1).reshape(L, H * dh).numpy(), atol=1e-12)


def test_attention_special_cases():
    r = _rng(5)
    H, dh = 2, 8
    v = r.normal(size=(5, H * dh))
    k = r.normal(size=(5, H * dh))
    # one key: the output is that key's value
    q1 = r.normal(size=(1, H * dh))
    assert np.allclose(O.attention(q1, k[:1], v[:1], H, dh), v[:1], atol=1e-14)
    # all-equal logits (q = 0): the mean of V
    q0 = np.zeros((2, H * dh))
    assert np.allclose(O.attention(q0, k, v, H, dh), np.repeat(v.mean(0, keepdims=True), 2, 0))
    # first causal row sees only key 0
    qq = r.normal(size=(5, H * dh))
    assert np.allclose(O.attention(qq, k, v, H, dh, causal=True)[0], v[0], atol=1e-14)


def _hf_rope(x, pos, H, dh, theta):
    from transformers import LlamaConfig
    from transformers.models.llama.modeling_llama import LlamaRotaryEmbedding, apply_rotary_pos_emb
    cfg = LlamaConfig(hidden_size=H * dh, num_attention_heads=H, head_dim=dh, rope_theta=theta,
                      max_position_embeddings=4096)
    emb = LlamaRotaryEmbedding(cfg)
    t = torch.from_numpy(x).view(1, len(pos), H, dh).transpose(1, 2)
    cos, sin = emb(t, torch.as_tensor(pos)[None, :])
    out, _ = apply_rotary_pos_emb(t, t, cos.double(), sin.double())
    return out.transpose(1, 2).reshape(len(pos), H * dh).numpy()


def test_rope_vs_transformers_and_invariants():
    r = _rng(6)
    H, dh, L = 2, 16, 9
    x = r.normal(size=(L, H * dh))
    pos = r.integers(0, 3000, size=L)
    got = O.rope(x, pos, H, dh, 10000.0)
    # transformers computes its angles in float32; allow for that
    assert np.allclose(got, _hf_rope(x, pos, H, dh, 10000.0), atol=2e-3)
    # position 0 is the identity
    assert np.array_equal(O.rope(x[:1], [0], H, dh, 10000.0), x[:1])
    # rotations preserve each (i, i + dh/2) pair's norm
    half = dh // 2
    xr = x.reshape(L, H, dh)
    gr = got.reshape(L, H, dh)
    assert np.allclose(xr[..., :half] ** 2 + xr[..., half:] ** 2,
                       gr[..., :half] ** 2 + gr[..., half:] ** 2, atol=1e-12)
    # rotations compose: rope(rope(x, m), n) == rope(x, m + n)
    m, n = 37, 1021
    a = O.rope(O.rope(x[:1], [m], H, dh, 10000.0), [n], H, dh, 10000.0)
    assert np.allclose(a, O.rope(x[:1], [m + n], H, dh, 10000.0), atol=1e-12)
    # q . k depends only on the offset between positions
    q, k = r.normal(size=(1, H * dh)), r.normal(size=(1, H * dh))
    d1 = (O.rope(q, [100], H, dh, 1e4) * O.rope(k, [70], H, dh, 1e4)).sum()
    d2 = (O.rope(q, [530], H, dh, 1e4) * O.rope(k, [500], H, dh, 1e4)).sum()
    assert abs(d1 - d2) < 1e-10


# --------------------------------------------------------------------------
# LoRA: closed forms and the merged / zero-rank invariants
# --------------------------------------------------------------------------
def test_lora_closed_form_unit_vectors():
    r = _rng(7)
    d_in, d_out, s = 12, 9, 2.0
    x = r.normal(size=(4, d_in))
    for i, j in [(0, 0), (3, 7), (11, 8)]:
        A = np.zeros((1, d_in)); A[0, i] = 1.0
        B = np.zeros((d_out, 1)); B[j, 0] = 1.0
        ref = np.zeros((4, d_out)); ref[:, j] = s * x[:, i]
        assert np.array_equal(O.lora_delta(x, A, B, s), ref)


def test_lora_merged_equals_unmerged_and_linear_in_scale():
    r = _rng(8)
    d_in, d_out, rk = 20, 14, 4
    x, W, A, B = (r.normal(size=sh) for sh in [(6, d_in), (d_out, d_in), (rk, d_in), (d_out, rk)])
    unmerged = O.linear(x, W) + O.lora_delta(x, A, B, 0.75)
    merged = O.linear(x, O.merged_adapter_weights(W, A, B, 0.75))
    assert np.allclose(unmerged, merged, rtol=0, atol=1e-12)
    assert np.allclose(O.lora_delta(x, A, B, 3.0), 4.0 * O.lora_delta(x, A, B, 0.75), atol=1e-12)


def _tiny(family, **kw):
    base = wl.WORKLOADS[1] if family == "encoder" else wl.WORKLOADS[4]
    args = dict(n_layers=1, d=32, n_heads=2, head_dim=16, d_ff=64, n_tasks=3, n_req=5,
                rank=4, dtype="f32", vocab=50)
    args.update(kw)
    return base.replace(**args)


def test_zero_rank_and_zero_b_equal_bare_backbone():
    for fam in ("encoder", "decoder"):
        w = _tiny(fam)
        W = oracle_weights(wl.backbone_layer(w, 0))
        ad = wl.adapters_layer(w, 0, ranks=np.array([0, 4, 4]))
        x = _rng(9).normal(size=(6, w.d))
        pos = np.arange(6)
        bare = O.layer(spec_of(w), W, None, x, pos=pos)[0]
        # rank 0: no adapter at all
        assert np.array_equal(O.layer(spec_of(w), W, oracle_adapter(ad, 0), x, pos=pos)[0], bare)
        # B = 0: the adapter adds exact zeros
        zb = {p: (a, np.zeros_like(b), s) for p, (a, b, s) in oracle_adapter(ad, 1).items()}
        assert np.array_equal(O.layer(spec_of(w), W, zb, x, pos=pos)[0], bare)
        # a real adapter changes the output
        assert not np.allclose(O.layer(spec_of(w), W, oracle_adapter(ad, 1), x, pos=pos)[0], bare)


# --------------------------------------------------------------------------
# whole layers vs library implementations
# --------------------------------------------------------------------------
def _torch_encoder_layer(w, W, merged=None):
    d = w.d
    m = torch.nn.TransformerEncoderLayer(d, w.n_heads, w.d_ff, dropout=0.0, activation="gelu",
                                         layer_norm_eps=w.norm_eps, batch_first=True,
                                         norm_first=True, dtype=torch.float64)
    wq = merged or {}
    qkv = np.concatenate([wq.get("q", W["w_qkv"][:d]), wq.get("k", W["w_qkv"][d:2 * d]),
                          wq.get("v", W["w_qkv"][2 * d:])])
    with torch.no_grad():
        m.self_attn.in_proj_weight.copy_(torch.from_numpy(qkv))
        m.self_attn.in_proj_bias.copy_(torch.from_numpy(W["b_qkv"]))
        m.self_attn.out_proj.weight.copy_(torch.from_numpy(wq.get("o", W["w_o"])))
        m.self_attn.out_proj.bias.copy_(torch.from_numpy(W["b_o"]))
        m.linear1.weight.copy_(torch.from_numpy(wq.get("up", W["w_up"])))
        m.linear1.bias.copy_(torch.from_numpy(W["b_up"]))
        m.linear2.weight.copy_(torch.from_numpy(wq.get("down", W["w_down"])))
        m.linear2.bias.copy_(torch.from_numpy(W["b_down"]))
        m.norm1.weight.copy_(torch.from_numpy(W["norm1_w"]))
        m.norm1.bias.copy_(torch.from_numpy(W["norm1_b"]))
        m.norm2.weight.copy_(torch.from_numpy(W["norm2_w"]))
        m.norm2.bias.copy_(torch.from_numpy(W["norm2_b"]))
    m.eval()
    return m


def _merged(W, adapter, d):
    base = {"q": W["w_qkv"][:d], "k": W["w_qkv"][d:2 * d], "v": W["w_qkv"][2 * d:],
            "o": W["w_o"], "gate": W.get("w_gate"), "up": W["w_up"], "down": W["w_down"]}
    return {p: O.merged_adapter_weights(base[p], A, B, s) for p, (A, B, s) in adapter.items()}


def test_encoder_layer_vs_torch_transformer_layer():
    w = _tiny("encoder", lora_targets=("q", "k", "v", "o", "up", "down"))
    W = oracle_weights(wl.backbone_layer(w, 0))
    ad = wl.adapters_layer(w, 0, b_std=0.3)
    x = _rng(10).normal(size=(9, w.d))
    with torch.no_grad():
        ref = _torch_encoder_layer(w, W)(torch.from_numpy(x)[None])[0].numpy()
        got = O.layer(spec_of(w), W, None, x)[0]
        assert np.allclose(got, ref, rtol=0, atol=1e-10)
        # with a task's adapter: torch's layer on the merged weights W + s B A
        a1 = oracle_adapter(ad, 1)
        ref = _torch_encoder_layer(w, W, _merged(W, a1, w.d))(torch.from_numpy(x)[None])[0].numpy()
        got = O.layer(spec_of(w), W, a1, x)[0]
        assert np.allclose(got, ref, rtol=0, atol=1e-10)


def _hf_llama_layer(w, W, merged=None):
    from transformers import LlamaConfig
    from transformers.models.llama.modeling_llama import LlamaDecoderLayer
    cfg = LlamaConfig(hidden_size=w.d, intermediate_size=w.d_ff, num_attention_heads=w.n_heads,
                      num_key_value_heads=w.n_heads, head_dim=w.head_dim, rms_norm_eps=w.norm_eps,
                      rope_theta=w.rope_theta, attention_bias=False, mlp_bias=False,
                      max_position_embeddings=4096)
    cfg._attn_implementation = "eager"
    m = LlamaDecoderLayer(cfg, layer_idx=0).double().eval()
    d = w.d
    wq = merged or {}
    with torch.no_grad():
        m.self_attn.q_proj.weight.copy_(torch.from_numpy(wq.get("q", W["w_qkv"][:d])))
        m.self_attn.k_proj.weight.copy_(torch.from_numpy(wq.get("k", W["w_qkv"][d:2 * d])))
        m.self_attn.v_proj.weight.copy_(torch.from_numpy(wq.get("v", W["w_qkv"][2 * d:])))
        m.self_attn.o_proj.weight.copy_(torch.from_numpy(wq.get("o", W["w_o"])))
        m.mlp.gate_proj.weight.copy_(torch.from_numpy(wq.get("gate", W["w_gate"])))
        m.mlp.up_proj.weight.copy_(torch.from_numpy(wq.get("up", W["w_up"])))
        m.mlp.down_proj.weight.copy_(torch.from_numpy(wq.get("down", W["w_down"])))
        m.input_layernorm.weight.copy_(torch.from_numpy(W["norm1_w"]))
        m.post_attention_layernorm.weight.copy_(torch.from_numpy(W["norm2_w"]))
    return m, cfg


def _run_hf(m, cfg, x, pos):
    from transformers.models.llama.modeling_llama import LlamaRotaryEmbedding
    L = x.shape[0]
    t = torch.from_numpy(x)[None]
    emb = LlamaRotaryEmbedding(cfg)
    pid = torch.as_tensor(pos)[None, :]
    cos, sin = emb(t, pid)
    mask = torch.triu(torch.full((L, L), float("-inf"), dtype=torch.float64), 1)[None, None]
    out = m(t, attention_mask=mask, position_ids=pid, position_embeddings=(cos.double(), sin.double()))
    out = out[0] if isinstance(out, tuple) else out
    return out[0].detach().numpy()


def test_decoder_layer_vs_transformers_llama_layer():
    w = _tiny("decoder")
    W = oracle_weights(wl.backbone_layer(w, 0))
    ad = wl.adapters_layer(w, 0, b_std=0.3)
    x = _rng(11).normal(size=(10, w.d))
    pos = np.arange(10)
    with torch.no_grad():
        m, cfg = _hf_llama_layer(w, W)
        ref = _run_hf(m, cfg, x, pos)
        got = O.layer(spec_of(w), W, None, x, pos=pos)[0]
        # transformers builds its rotary angles in float32
        assert O.row_rel_error(got, ref) < 1e-5
        a2 = oracle_adapter(ad, 2)
        m, cfg = _hf_llama_layer(w, W, _merged(W, a2, w.d))
        ref = _run_hf(m, cfg, x, pos)
        got = O.layer(spec_of(w), W, a2, x, pos=pos)[0]
        assert O.row_rel_error(got, ref) < 1e-5


def test_decode_step_equals_last_prefill_row():
    w = _tiny("decoder")
    W = oracle_weights(wl.backbone_layer(w, 0))
    ad = oracle_adapter(wl.adapters_layer(w, 0, b_std=0.3), 1)
    L = 12
    x = _rng(12).normal(size=(L + 1, w.d))
    full, k, v = O.layer(spec_of(w), W, ad, x, pos=np.arange(L + 1))
    step, k1, v1 = O.layer(spec_of(w), W, ad, x[L:], pos=[L], kv=(k[:L], v[:L]))
    assert np.allclose(step, full[L:], rtol=0, atol=1e-12)
    assert np.allclose(k1, k[L:], atol=1e-12) and np.allclose(v1, v[L:], atol=1e-12)


@pytest.mark.parametrize("L,m", [(12, 5), (7, 1), (1, 9), (20, 13)])
def test_prefill_chunk_equals_rows_of_full_prefill(L, m):
    """A prompt chunk of m rows after L cached tokens (the chunked-prefill
    step) equals rows L .. L+m-1 of the whole (L+m)-token prefill: each chunk
    row attends causally to the cached keys and the chunk's earlier rows.
    Pins the multi-row branch of the cached-key attention (q_offset > 0,
    causal mask inside the chunk), not only its one-row decode case."""
    w = _tiny("decoder")
    W = oracle_weights(wl.backbone_layer(w, 0))
    ad = oracle_adapter(wl.adapters_layer(w, 0, b_std=0.3), 2)
    x = _rng(40 + L + m).normal(size=(L + m, w.d))
    full, k, v = O.layer(spec_of(w), W, ad, x, pos=np.arange(L + m))
    chunk, kc, vc = O.layer(spec_of(w), W, ad, x[L:], pos=np.arange(L, L + m), kv=(k[:L], v[:L]))
    assert np.abs(chunk - full[L:]).max() <= 1e-12 * np.abs(full[L:]).max()
    assert np.abs(kc - k[L:]).max() <= 1e-12 * np.abs(k[L:]).max()
    assert np.abs(vc - v[L:]).max() <= 1e-12 * np.abs(v[L:]).max()
    # a wrong mask inside the chunk (every chunk row seeing the whole chunk) is caught
    q_full = O.rope(O.linear(O.rms_norm(x, W["norm1_w"], w.norm_eps), W["w_qkv"][:w.d]),
                    np.arange(L + m), w.n_heads, w.head_dim, w.rope_theta)
    if m > 1:
        leak = O.attention(q_full[L:], k, v, w.n_heads, w.head_dim, causal=False)
        ok = O.attention(q_full[L:], k, v, w.n_heads, w.head_dim, causal=True, q_offset=L)
        assert np.abs(leak - ok).max() > 1e-3


# --------------------------------------------------------------------------
# the method's re-association equals the per-request definition
# --------------------------------------------------------------------------
@pytest.mark.parametrize("family", ["encoder", "decoder"])
def test_batched_equals_per_request_and_isolation(family):
    w = _tiny(family, n_tasks=4, lora_targets=wl.PROJ)
    W = oracle_weights(wl.backbone_layer(w, 0))
    ranks = np.array([4, 0, 8, 4])
    ad = wl.adapters_layer(w, 0, ranks=ranks, b_std=0.3)
    per_task = [oracle_adapter(ad, t) for t in range(w.n_tasks)]
    task_id = np.array([2, 0, 2, 3, 0, 1, 2])
    lens = np.array([3, 5, 1, 4, 2, 6, 3])
    pl = O.plan(task_id, lens, w.n_tasks)
    r = _rng(13)
    x_orig = r.normal(size=(int(lens.sum()), w.d))
    cu_o = pl["cu_orig"]
    rows = np.concatenate([x_orig[cu_o[i]:cu_o[i + 1]] for i in pl["order"]])
    got = O.batched_layer(spec_of(w), W, per_task, rows, pl)
    for p, i in enumerate(pl["order"]):
        xi = x_orig[cu_o[i]:cu_o[i + 1]]
        ref = O.layer(spec_of(w), W, per_task[task_id[i]], xi, pos=np.arange(len(xi)))[0]
        seg = got[pl["cu_seqlens"][p]:pl["cu_seqlens"][p + 1]]
        assert np.allclose(seg, ref, rtol=0, atol=1e-12)
    # isolation: replacing task 3's adapter leaves every other task's rows unchanged
    other = list(per_task)
    other[3] = {k: (a, 5 * b, s) for k, (a, b, s) in per_task[3].items()}
    got2 = O.batched_layer(spec_of(w), W, other, rows, pl)
    mask = np.repeat(pl["task"] != 3, lens[pl["order"]])
    assert np.array_equal(got2[mask], got[mask])
    assert not np.allclose(got2[~mask], got[~mask])


def test_head_identity_and_pooling():
    r = _rng(14)
    xn = r.normal(size=(5, 6))
    assert np.array_equal(O.pool(xn, "first"), xn[0])
    assert np.array_equal(O.pool(xn, "last"), xn[-1])
    assert np.allclose(O.pool(xn, "mean"), xn.sum(0) / 5)
    p = r.normal(size=6)
    assert np.array_equal(O.head(p, np.eye(6), np.zeros(6)), p)
    Wt, bt = r.normal(size=(3, 6)), r.normal(size=3)
    ref = np.array([sum(Wt[j, c] * p[c] for c in range(6)) + bt[j] for j in range(3)])
    assert np.allclose(O.head(p, Wt, bt), ref, atol=1e-13)


def test_row_rel_error_measure():
    ref = np.array([[1.0, -4.0], [0.0, 0.0]])
    got = np.array([[1.2, -4.0], [0.0, 0.5]])
    assert O.row_rel_error(got, ref) == pytest.approx(0.5)
    assert O.row_rel_error(ref, ref) == 0.0


def test_mlp_head_pins():
    """Two-layer MLP decoder head: a worked example with the standard normal
    CDF values Phi(3) = 0.9986501, Phi(-1) = 0.1586553, and the reduction to
    the linear head (identity first layer, ReLU, non-negative input)."""
    pooled = np.array([1.0, -2.0])
    W1 = np.array([[1.0, 1.0], [2.0, 0.0]])
    b1 = np.array([0.0, 1.0])
    W = np.array([[1.0, 2.0]])
    b = np.array([0.5])
    # pre-activation [-1, 3]
    assert np.allclose(O.head_mlp(pooled, W1, b1, W, b, act="relu"), [0.0 + 2 * 3.0 + 0.5])
    assert np.allclose(O.head_mlp(pooled, W1, b1, W, b, act="gelu"),
                       [-1 * 0.1586553 + 2 * 3 * 0.9986501 + 0.5], atol=1e-6)
    rng = np.random.default_rng(0)
    x = np.abs(rng.normal(size=16))
    W2 = rng.normal(size=(5, 16))
    b2 = rng.normal(size=5)
    assert np.allclose(O.head_mlp(x, np.eye(16), np.zeros(16), W2, b2, act="relu"), O.head(x, W2, b2))


def test_channel_combiner_pins():
    """Linear channel combiner (C channels to one) and the patch embedding it
    feeds: a hand-worked example, selection of one channel by a unit weight,
    the channel mean, and patches cut in order."""
    x = np.array([[1.0, 2.0], [3.0, 4.0], [5.0, 6.0]])          # 3 channels, 2 samples
    assert np.allclose(O.channel_combine(x, [1.0, 0.0, -1.0], 0.5), [1 - 5 + 0.5, 2 - 6 + 0.5])
    assert np.allclose(O.channel_combine(x, [0.0, 1.0, 0.0]), x[1])
    assert np.allclose(O.channel_combine(x, [1 / 3] * 3), [3.0, 4.0])
    assert np.allclose(O.channel_combine(x, [2.0, 0.0, 0.0], np.array([1.0])), [3.0, 5.0])
    s = np.arange(6.0)                                          # two patches of 3
    W_pe = np.array([[1.0, 0.0, 0.0], [0.0, 0.0, 1.0]])
    assert np.allclose(O.patch_embed(s, 3, W_pe, np.array([0.0, 10.0])), [[0.0, 12.0], [3.0, 15.0]])
