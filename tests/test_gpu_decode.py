"""Parity of moba_decode (one new query per sequence against its key/value
cache) with the oracle, through the C ABI.

The decode query of sequence s sits at the last cached position, so its
result is the last row of the prefill over the cache: the oracle's gate and
attention for the rows (cu[s+1] - 1, h), reading only those rows' query
vectors.  MoBA mode with the block means passed in and computed on the fly,
and full-attention mode (what the paper uses for generation).

The decode gate sums scores in fp32 in its own fixed order; a row whose
(k-1)-th and k-th best oracle scores are closer than the gate's rounding
bound (tau of tests/parity.py) has more than one correct selection, and its
output is compared with the oracle's attention over the admissible selection
closest to it (parity.check_rows_any_selection); no row is left out.
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


CASES = [
    # seqlens, hq, hkv, B, topk
    ((300,), 2, 2, 64, 3),
    ((1000, 1, 517), 4, 2, 128, 3),
    ((777,), 8, 2, 100, 4),
    ((513, 129, 64), 4, 1, 48, 5),
    ((700,), 4, 4, 96, 20),
    ((2048, 333), 16, 2, 256, 3),
    ((5000,), 4, 1, 1000, 2),
    ((333, 1), 2, 1, 7, 6),
    ((4097, 4096, 300), 8, 2, 512, 4),
    ((600, 45), 16, 1, 64, 3),   # the largest group decode takes
    ((50, 2), 2, 1, 1, 5),       # one-key blocks
    ((24000, 300), 4, 1, 4096, 5),  # combine in two shares per row (80 MoBA / 94 full slots)
    ((1025, 1026), 2, 1, 1, 4),  # 1024 past blocks (the most the gate ranks in parallel), then 1025
    ((2600,), 2, 1, 2, 6),       # 1299 past blocks: the gate's argmax rounds
    ((900,), 16, 1, 16, 24),     # 16 x 24 selections per group: the block union takes two passes
]


def decode_case(seqlens, hq, hkv, B, seed):
    q, k, v, cu = inputs.make(seqlens, hq, hkv, 128, torch.bfloat16, B, 0.5, seed, device=DEV)
    last = (cu[1:] - 1).to(torch.int64)
    qd = q[last.to(DEV)].contiguous()  # the new token of each sequence
    return q, qd, k, v, cu


@pytest.mark.parametrize("seqlens,hq,hkv,B,topk", CASES,
                         ids=["-".join(map(str, c[0])) + "_h%dx%d_B%d_k%d" % c[1:] for c in CASES])
@pytest.mark.parametrize("mode", ["moba_kbar", "moba", "full"])
def test_decode(seqlens, hq, hkv, B, topk, mode):
    seed = sum(seqlens) + B + 3
    q, qd, k, v, cu = decode_case(seqlens, hq, hkv, B, seed)
    T = q.shape[0]
    S = len(seqlens)
    kbar = binding.pool(k, cu, B) if mode == "moba_kbar" else None
    out, lse = binding.decode(qd, k, v, cu, B, 0 if mode == "full" else topk, kbar=kbar)
    torch.cuda.synchronize()
    rows = np.array([(int(cu[s + 1]) - 1) * hq + h for s in range(S) for h in range(hq)], np.int64)
    q_rows = inputs.to_oracle(qd.reshape(S * hq, 128))
    kn, vn = inputs.to_oracle(k), inputs.to_oracle(v)
    cun = cu.numpy()
    gout = out.float().cpu().numpy().reshape(S * hq, 128)
    glse = lse.cpu().numpy().T.reshape(S * hq)
    if mode == "full":
        Bf = max(seqlens)
        sel = np.zeros((len(rows), 1), np.int32)
        oout, olse = oracle.attend_rows(q_rows, T, hq, kn, vn, cun, Bf, sel, rows)
        mx, mean, lmx = parity.compare_outputs(gout, glse, oout, olse, "bf16", mode)
        multi = other = 0
    else:
        mx, mean, lmx, multi, other = parity.check_rows_any_selection(
            gout, glse, q_rows, rows, T, hq, kn, vn, cun, B, topk, mode)
    print("%s rows %d (several admissible selections %d, matched another %d) out max-abs %.2e "
          "mean-abs %.2e lse %.2e" % (mode, len(rows), multi, other, mx, mean, lmx))


def test_decode_matches_prefill_last_rows():
    """On a cache whose rows have no near ties, decode equals the prefill's
    last row within bf16 rounding (the two paths round differently)."""
    q, qd, k, v, cu = decode_case((3000, 1500), 8, 2, 256, 77)
    out_p, lse_p = binding.forward(q, k, v, cu, 256, 4)
    out_d, lse_d = binding.decode(qd, k, v, cu, 256, 4)
    torch.cuda.synchronize()
    last = (cu[1:] - 1).to(torch.int64).to(DEV)
    assert (out_p[last].float() - out_d.float()).abs().max().item() <= 2e-2
    assert (lse_p[:, last] - lse_d).abs().max().item() <= 1e-3


def test_decode_rejects_empty_sequence():
    q, qd, k, v, cu = decode_case((100, 50), 2, 1, 32, 5)
    bad = torch.tensor([0, 150, 150], dtype=torch.int32)
    with pytest.raises(binding.MobaError) as e:
        binding.decode(qd, k, v, bad, 32, 2)
    assert e.value.name == "MOBA_ERR_SEQLENS"
