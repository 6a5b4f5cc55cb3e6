"""Decode parity at full workload sizes, in the launch configuration that
`bench.py --decode` times: the workload's whole cache, one new query per
sequence (the last token's), the cache's block means computed once by
moba_pool and passed in, then one moba_decode call in full-attention mode and
one in MoBA mode.

Every decode row is checked (S * Hq rows): the oracle computes the last
prefill row of each sequence from that row's query vector alone, over up to
the whole 1M-token cache in full mode.  A MoBA row whose (k-1)-th and k-th
oracle gate scores lie within the gate's rounding bound has more than one
correct selection; it is compared with the oracle's attention over the
admissible selection closest to it (parity.check_rows_any_selection), so no
row is left out.  The tolerances are those of tests/parity.py.
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
    mmx, mmean, mlmx, multi, other = parity.check_rows_any_selection(
        got["moba"][0], got["moba"][1], q_rows, rows, T, Hq, kn, vn, cun, w.block_size, w.topk,
        "moba")
    print("%s: %d decode rows; full out max-abs %.2e mean-abs %.2e lse %.2e; MoBA (rows with "
          "several admissible selections %d, matched another %d) out max-abs %.2e mean-abs %.2e "
          "lse %.2e" % (name, len(rows), fmx, fmean, flmx, multi, other, mmx, mmean, mlmx))
