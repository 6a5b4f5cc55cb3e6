"""Parity at the full sizes of the five prefill workloads, in the launch
configuration the benchmark times (one moba_forward call over the batch).

The selection is compared with the oracle's on every row of every workload
(at 1M tokens four query heads at a time, about a minute of host time), and
the selection invariants are checked on every row on the GPU.  Outputs are
compared on every row where the oracle finishes in seconds (the 1K fp32 and
8K workloads), otherwise on a fixed sample: for each query head the
block-boundary positions, 64 seeded uniform positions, and the whole last
block of one head.
"""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2502_13189_amd import binding, inputs
import parity

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.load()


def gpu_selection_invariants(sel, cu, B, topk):
    """On every row: the current block c is selected, nothing after it, the
    history part is strictly ascending below c with min(topk-1, c) entries,
    and the rest is -1 padding."""
    T, Hq, K = sel.shape
    cu_d = cu.to(sel.device, torch.int64)
    t = torch.arange(T, device=sel.device)
    s = torch.searchsorted(cu_d, t, right=True) - 1
    c = ((t - cu_d[s]) // B)[:, None].expand(T, Hq)
    nh = torch.clamp(c, max=topk - 1)
    idx = torch.arange(K, device=sel.device)[None, None, :]
    s64 = sel.to(torch.int64)
    cur = torch.gather(s64, 2, nh[..., None])[..., 0]
    assert torch.equal(cur, c)
    hist = idx < nh[..., None]
    assert bool(((s64 < c[..., None]) | ~hist).all())
    assert bool(((s64 >= 0) | ~hist).all())
    if K > 1:
        inc = (s64[..., 1:] > s64[..., :-1]) | ~hist[..., 1:]
        assert bool(inc.all())
    pad = idx > nh[..., None]
    assert bool(((s64 == -1) | ~pad).all())


def run_workload(name, out_rows="all", head_chunk=32):
    w = inputs.WORKLOADS[name]
    q, k, v, cu = inputs.make_workload(w, device=DEV)
    T, Hq = q.shape[0], q.shape[1]
    dtype = w.dtype
    out, lse = binding.forward(q, k, v, cu, w.block_size, w.topk)
    sel = binding.select(q, k, cu, w.block_size, w.topk)
    torch.cuda.synchronize()
    gpu_selection_invariants(sel, cu, w.block_size, w.topk)
    qn, kn, vn = parity.host_inputs(q, k, v)
    cun = cu.numpy()
    # every row's selection, in chunks of query heads (bounded host memory)
    pooled = oracle.pool(kn, cun, w.block_size, with_abs=True)
    nsel, nbad = 0, 0
    for h0 in range(0, Hq, head_chunk):
        heads = np.arange(h0, min(Hq, h0 + head_chunk))
        srows = (np.arange(T, dtype=np.int64)[:, None] * Hq + heads[None, :]).ravel()
        gsel = sel.view(T * Hq, w.topk)[torch.as_tensor(srows, device=DEV)].cpu().numpy()
        _, bad = parity.check_selection(gsel, srows, qn, kn, cun, w.block_size, w.topk,
                                        exact=(dtype == "f32"), pooled=pooled)
        nsel += len(srows)
        nbad += len(bad)
        del gsel
        print("[wl] %s: selection of heads %d-%d compared (tie-explained %d)"
              % (name, heads[0], heads[-1], len(bad)), flush=True)
    assert nsel == T * Hq
    orows = np.arange(T * Hq, dtype=np.int64) if out_rows == "all" else \
        inputs.sample_rows(w, full_heads=(0,))
    # the selection used for the output check: the oracle's, except on
    # tie-explained rows, where the GPU's own selection is used
    ogsel = sel.view(T * Hq, w.topk)[torch.as_tensor(orows, device=DEV)].cpu().numpy()
    oosel = oracle.select(qn, pooled[0], cun, w.block_size, w.topk, rows=orows)
    diff = (ogsel != oosel).any(axis=1)
    if diff.any():
        parity.check_selection(ogsel[diff], orows[diff], qn, kn, cun, w.block_size, w.topk,
                               exact=(dtype == "f32"), pooled=pooled)
    use = np.where(diff[:, None], ogsel, oosel)
    oout, olse = oracle.attend(qn, kn, vn, cun, w.block_size, use, rows=orows)
    gout, glse = parity.gather_rows(out, lse, orows)
    mx, mean, lmx = parity.compare_outputs(gout, glse, oout, olse, dtype, name)
    print("%s: selection rows %d (tie-explained %d), output rows %d, max-abs %.2e mean-abs %.2e "
          "lse %.2e" % (name, nsel, nbad, len(orows), mx, mean, lmx))
    return q, k, v, cu


def test_f32_L1k():
    run_workload("f32_L1k_h1_B128_k3")


def test_bf16_L8k_mha():
    run_workload("bf16_L8k_mha32_B512_k3")


def test_bf16_L32k_gqa():
    run_workload("bf16_L32k_gqa32x8_B2048_k3", out_rows="sample")


def test_bf16_varlen4():
    run_workload("bf16_varlen4_T111920_mha32_B1024_k4", out_rows="sample")


def test_bf16_L1M_gqa():
    q, k, v, cu = run_workload("bf16_L1M_gqa32x8_B4096_k12", out_rows="sample", head_chunk=4)
    del q, k, v
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["f32_L1k_h1_B128_k3", "bf16_L8k_mha32_B512_k3"])
def test_dense_workload(name):
    w = inputs.WORKLOADS[name]
    q, k, v, cu = inputs.make_workload(w, device=DEV)
    rows = None if w.dtype == "f32" else inputs.sample_rows(w, full_heads=(0,))
    parity.dense_parity(q, k, v, cu, rows=rows, dtype=w.dtype)
