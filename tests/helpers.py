"""Test-side glue: turns drawn workload tensors into the oracle's float64 inputs."""
import numpy as np
import torch

from paper_2606_09643_amd import workloads as wl


def np64(t):
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        return t.astype(np.float64)
    return t.detach().to("cpu", torch.float64).numpy()


def spec_of(w):
    return {"family": w.family, "n_heads": w.n_heads, "head_dim": w.head_dim,
            "norm": w.norm, "eps": w.norm_eps, "rope_theta": w.rope_theta}


def oracle_weights(W):
    return {k: np64(v) for k, v in W.items()}


def oracle_adapter(ad, t):
    """{proj: (A, B, scale)} of task t, or None when its rank is 0."""
    if ad is None or int(ad.rank[t]) == 0:
        return None
    return {p: (np64(ad.a(p, t)), np64(ad.b(p, t)), float(ad.scale[t])) for p in ad.A}
