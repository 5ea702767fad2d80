"""Shared pieces of the GPU parity tests: oracle evaluation over a plan-ordered
batch, and tolerances.  Imports the oracle (test infrastructure) and the
product binding side by side; neither imports the other."""
import numpy as np
import torch

from oracle import vfm_oracle as O
from paper_2606_09643_amd import runner as R
from paper_2606_09643_amd import workloads as wl
from tests.helpers import np64, oracle_adapter, oracle_weights, spec_of

TOL = {"bf16": 2e-2, "f32": 1e-5}


def tol(w):
    return TOL[w.dtype]


def log(msg):
    print(msg, flush=True)


def oracle_plan(w, batch, n_out=None):
    return O.plan(batch.task_id, batch.seq_len, w.n_tasks,
                  ctx=batch.ctx if w.mode == "decode" else None, n_out=n_out)


def expected_embed(w, batch, inp, pl):
    """Input rows in plan order (float64), from the oracle's plan."""
    cu_o = pl["cu_orig"]
    if inp.mode == 0:
        src = np64(inp.src)
    elif inp.mode == 1:
        ids = inp.src.cpu().numpy()
        src = np64(inp.table)[ids]
    else:
        src = O.linear(np64(inp.src), np64(inp.table), np64(inp.bias))
    return np.concatenate([src[cu_o[i]:cu_o[i + 1]] for i in pl["order"]])


def as_f32(rows):
    """fp64 rows rounded to fp32 (the GPU residual stream's type), as fp64:
    the values both sides start from when a GPU call is fed oracle rows."""
    return np.asarray(rows, np.float64).astype(np.float32).astype(np.float64)


def set_rows(x_dev, rows, r0=0):
    """Writes oracle-side rows (plan order, from row r0) into the GPU's fp32
    residual stream, so a GPU call and the oracle take the same input and no
    oracle input comes from the GPU path."""
    t = torch.from_numpy(np.ascontiguousarray(rows, np.float32)).to(x_dev.device)
    x_dev[r0:r0 + t.shape[0]].copy_(t)


def seeded_rows(n, d, seed):
    """Standard normal rows from a seeded host generator, rounded to fp32."""
    return as_f32(np.random.default_rng(seed).standard_normal((n, d)))


def oracle_layer_rows(w, W_np, ad, pl, x_plan, reqs, kv=None, li=0):
    """Oracle layer for the chosen plan positions; returns {p: (y, k, v)}.
    kv: the decode KV cache (layer li's cached keys are read from it)."""
    spec = spec_of(w)
    cu = pl["cu_seqlens"]
    res = {}
    for p in reqs:
        sl = slice(int(cu[p]), int(cu[p + 1]))
        t = int(pl["task"][p])
        kvp = None
        if kv is not None:
            i = int(pl["order"][p])
            c = int(pl["pos"][sl][0])
            kr, vr = kv.rows(li, int(kv.kv_start[i]), c)
            kvp = (np64(kr), np64(vr))
        res[p] = O.layer(spec, W_np, oracle_adapter(ad, t), x_plan[sl], pos=pl["pos"][sl], kv=kvp)
    return res


def oracle_heads(w, model, pl, x_plan, n_out):
    """Final norm, pooling and head per request, in original order (list)."""
    spec = spec_of(w)
    fw, fb = np64(model.final["w"]), np64(model.final["b"])
    cu = pl["cu_seqlens"]
    outs = [None] * len(pl["order"])
    for p, i in enumerate(pl["order"]):
        xn = O.final(spec, fw, fb, x_plan[int(cu[p]):int(cu[p + 1])])
        t = int(pl["task"][p])
        pooled = O.pool(xn, w.pool)
        outs[i] = O.head(pooled, np64(model.heads.W[t]), np64(model.heads.b[t]))
    return outs


def pick_requests(pl, k=6):
    """A deterministic spread of plan positions: first / last of the largest
    and smallest segments, segment boundaries, shortest and longest."""
    n = len(pl["order"])
    if n <= k:
        return list(range(n))
    seg = pl["seg_req"]
    sizes = np.diff(seg)
    nz = np.nonzero(sizes)[0]
    big, small = nz[np.argmax(sizes[nz])], nz[np.argmin(sizes[nz])]
    lens = np.diff(pl["cu_seqlens"])
    cand = [seg[big], seg[big + 1] - 1, seg[small], int(np.argmin(lens)), int(np.argmax(lens)),
            0, n - 1]
    out = []
    for c in cand:
        if int(c) not in out:
            out.append(int(c))
    return out[:k]
