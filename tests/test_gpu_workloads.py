"""Parity at the full sizes of the five prefill workloads, in the launch
configuration the benchmark times (one moba_forward call over the batch).

Every row is compared where the oracle finishes in seconds (the 1K fp32 and
8K workloads).  Otherwise the selection is compared on every row (32K and the
packed batch) or on every row of two query heads (1M), the selection
invariants are checked on every row on the GPU, and outputs are compared on a
fixed sample: for each query head the block-boundary positions, 64 seeded
uniform positions, and the whole last block of one head.
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


def run_workload(name, sel_rows="all", out_rows="all"):
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
    if sel_rows == "all":
        srows = np.arange(T * Hq, dtype=np.int64)
    else:
        heads = sel_rows
        srows = (np.arange(T, dtype=np.int64)[:, None] * Hq + np.array(heads)[None, :]).ravel()
    gsel = sel.view(T * Hq, w.topk)[torch.as_tensor(srows, device=DEV)].cpu().numpy()
    osel, bad = parity.check_selection(gsel, srows, qn, kn, cun, w.block_size, w.topk,
                                       exact=(dtype == "f32"))
    orows = srows if out_rows == "all" else inputs.sample_rows(w, full_heads=(0,))
    # the selection used for the output check: the oracle's, except on
    # tie-explained rows, where the GPU's own selection is used
    ogsel = sel.view(T * Hq, w.topk)[torch.as_tensor(orows, device=DEV)].cpu().numpy()
    oosel = oracle.select(qn, oracle.pool(kn, cun, w.block_size), cun, w.block_size, w.topk,
                          rows=orows)
    diff = (ogsel != oosel).any(axis=1)
    if diff.any():
        parity.check_selection(ogsel[diff], orows[diff], qn, kn, cun, w.block_size, w.topk,
                               exact=(dtype == "f32"))
    use = np.where(diff[:, None], ogsel, oosel)
    oout, olse = oracle.attend(qn, kn, vn, cun, w.block_size, use, rows=orows)
    gout, glse = parity.gather_rows(out, lse, orows)
    mx, mean, lmx = parity.compare_outputs(gout, glse, oout, olse, dtype, name)
    print("%s: selection rows %d (tie-explained %d), output rows %d, max-abs %.2e mean-abs %.2e "
          "lse %.2e" % (name, len(srows), len(bad), len(orows), mx, mean, lmx))
    return q, k, v, cu


def test_f32_L1k():
    run_workload("f32_L1k_h1_B128_k3")


def test_bf16_L8k_mha():
    run_workload("bf16_L8k_mha32_B512_k3")


def test_bf16_L32k_gqa():
    run_workload("bf16_L32k_gqa32x8_B2048_k3", sel_rows="all", out_rows="sample")


def test_bf16_varlen4():
    run_workload("bf16_varlen4_T111920_mha32_B1024_k4", sel_rows="all", out_rows="sample")


def test_bf16_L1M_gqa():
    q, k, v, cu = run_workload("bf16_L1M_gqa32x8_B4096_k12", sel_rows=[0, 31], out_rows="sample")
    del q, k, v
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["f32_L1k_h1_B128_k3", "bf16_L8k_mha32_B512_k3"])
def test_dense_workload(name):
    w = inputs.WORKLOADS[name]
    q, k, v, cu = inputs.make_workload(w, device=DEV)
    rows = None if w.dtype == "f32" else inputs.sample_rows(w, full_heads=(0,))
    parity.dense_parity(q, k, v, cu, rows=rows, dtype=w.dtype)
