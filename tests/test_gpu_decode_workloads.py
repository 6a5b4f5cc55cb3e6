"""Decode parity at full workload sizes, in the launch configuration that
`bench.py --decode` times: the workload's whole cache, one new query per
sequence (the last token's), the cache's block means computed once by
moba_pool and passed in, then one moba_decode call in full-attention mode and
one in MoBA mode.

Every decode row is checked (S * Hq rows): the oracle computes the last
prefill row of each sequence from that row's query vector alone, over up to
the whole 1M-token cache in full mode.  MoBA rows whose k-th and (k+1)-th
oracle gate scores lie within the gate's rounding bound have two correct
selections and are skipped (counted); the tolerances are those of
tests/parity.py.
"""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2502_13189_amd import binding, inputs
import parity

pytestmark = pytest.mark.gpu
DEV = "cuda:0"

WORKLOADS = ["bf16_L1M_gqa32x8_B4096_k12", "bf16_varlen4_T111920_mha32_B1024_k4"]


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.load()


@pytest.mark.parametrize("name", WORKLOADS)
def test_decode_workload(name):
    w = inputs.WORKLOADS[name]
    print("[dec] %s: generating" % name, flush=True)
    q, k, v, cu = inputs.make_workload(w, device=DEV)
    T, Hq, D = q.shape
    S = len(w.seqlens)
    last = (cu[1:] - 1).to(torch.int64).to(DEV)
    qd = q[last].contiguous()
    del q
    kbar = binding.pool(k, cu, w.block_size)
    got = {}
    for mode, kk in (("full", 0), ("moba", w.topk)):
        out, lse = binding.decode(qd, k, v, cu, w.block_size, kk, kbar=kbar)
        torch.cuda.synchronize()
        got[mode] = (out.float().cpu().numpy().reshape(S * Hq, D), lse.cpu().numpy().T.reshape(S * Hq))
    q_rows = inputs.to_oracle(qd.reshape(S * Hq, D))
    del qd, kbar
    kn, vn = inputs.to_oracle(k), inputs.to_oracle(v)
    del k, v
    torch.cuda.empty_cache()
    cun = cu.numpy()
    rows = np.array([(int(cun[s + 1]) - 1) * Hq + h for s in range(S) for h in range(Hq)], np.int64)

    print("[dec] %s: oracle, full attention over every cached key" % name, flush=True)
    sel0 = np.zeros((len(rows), 1), np.int32)
    oout, olse = oracle.attend_rows(q_rows, T, Hq, kn, vn, cun, max(w.seqlens), sel0, rows)
    gout, glse = got["full"]
    fmx, fmean, flmx = parity.compare_outputs(gout, glse, oout, olse, "bf16", "full")

    print("[dec] %s: oracle, MoBA gate and attention" % name, flush=True)
    osel, amb = parity.decode_ambiguous_rows(q_rows, rows, T, Hq, kn, cun, w.block_size, w.topk)
    oout, olse = oracle.attend_rows(q_rows, T, Hq, kn, vn, cun, w.block_size, osel, rows)
    keep = ~amb
    gout, glse = got["moba"]
    mmx, mmean, mlmx = parity.compare_outputs(gout[keep], glse[keep], oout[keep], olse[keep], "bf16",
                                              "moba")
    print("%s: %d decode rows; full out max-abs %.2e mean-abs %.2e lse %.2e; MoBA (near-tie rows "
          "skipped %d) out max-abs %.2e mean-abs %.2e lse %.2e"
          % (name, len(rows), fmx, fmean, flmx, int(amb.sum()), mmx, mmean, mlmx))
    assert keep.sum() >= len(rows) // 2, "most rows must be unambiguous"
