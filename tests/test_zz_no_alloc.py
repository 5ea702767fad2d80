"""The allocation-free layer call (vfm_layer_forward_noalloc) against the
workspace-taking one (vfm_layer_forward), through the C ABI: two calls in a
row on each path, the second with a smaller batch, every output compared
bit for bit (same kernels, same summation orders), including the K / V rows
a decode step writes.  Batches whose workspace exceeds the library's fixed
scratch array are refused on the host."""
import numpy as np
import pytest
import torch

from paper_2606_09643_amd import binding as B
from paper_2606_09643_amd import runner as R
from paper_2606_09643_amd import workloads as wl
from tests.gpu_common import log

pytestmark = pytest.mark.gpu


def _run_both(w, model, batch):
    """One layer over `batch` on both entry points (separate inputs and
    caches holding the same values); returns, per output, whether the two
    are bit-identical."""
    kv_a = R.KVCache(w, batch, 1) if w.mode == "decode" else None
    kv_b = R.KVCache(w, batch, 1) if w.mode == "decode" else None
    pb = R.make_batch(w, batch, model.heads, kv_a)
    inp = R.Inputs(w, batch)
    fa = R.Forward(model, pb, inp, kv_a)
    fa.embed()
    x_b = fa.x.clone()
    log(f"  {w.name}: T={pb.T}, workspace {fa.ws.numel() / 2**20:.1f} MiB "
        f"(scratch {B.VFM_NOALLOC_SCRATCH_BYTES / 2**20:.0f} MiB)")
    fa.layer(0)
    kc = kv_b.k[0] if kv_b is not None else None
    vc = kv_b.v[0] if kv_b is not None else None
    slots = kv_b.slots if kv_b is not None else 0
    B.vfm_layer_forward_noalloc(model.cfg, model.c_layers[0], model.lora_c(0), pb.c, x_b, kc, vc, slots)
    torch.cuda.synchronize()
    same = {"x": torch.equal(fa.x, x_b)}
    if kv_a is not None:
        same["k"] = torch.equal(kv_a.k[0], kv_b.k[0])
        same["v"] = torch.equal(kv_a.v[0], kv_b.v[0])
    del fa, kv_a, kv_b, x_b
    torch.cuda.empty_cache()
    return same


@pytest.mark.parametrize("idx,small", [
    (5, dict(task_id=[7, 0, 7, 127, 3, 0, 64] * 6, ctx=[0, 1, 1023, 1024, 2048, 300, 77] * 6)),
    (2, dict(task_id=[5, 0, 5, 2, 9, 0, 15], seq_len=[197] * 7)),
])
def test_noalloc_layer_matches_workspace_layer(idx, small):
    w = wl.WORKLOADS[idx]
    model = R.Model(w, n_layers=1)
    big = wl.draw_batch(w)
    n = len(small["task_id"])
    seq = small.get("seq_len", [1] * n)
    little = wl.Batch(np.asarray(small["task_id"], np.int32), np.asarray(seq, np.int32),
                      np.asarray(small["ctx"], np.int32) if "ctx" in small else None)
    assert little.total_rows < big.total_rows
    for name, batch in (("full batch", big), ("smaller batch", little)):
        log(f"workload {idx} {name}")
        for key, same in _run_both(w, model, batch).items():
            assert same, f"{name}: {key} differs"


def test_noalloc_refuses_batches_beyond_the_scratch_array():
    """The 7B prefill batch needs a ~705 MiB workspace, beyond the fixed
    array: refused with VFM_ERR_WORKSPACE before anything is launched."""
    w = wl.WORKLOADS[4]
    model = R.Model(w, n_layers=1)
    batch = wl.draw_batch(w)
    pb = R.make_batch(w, batch, None)
    x = torch.zeros(pb.T, w.d, dtype=torch.float32, device="cuda")
    with pytest.raises(B.VfmError) as e:
        B.vfm_layer_forward_noalloc(model.cfg, model.c_layers[0], model.lora_c(0), pb.c, x)
    assert e.value.status == B.VFM_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert not x.any()
