"""Parity on seeded random shapes, beyond the hand-picked cases: ragged
sequence mixes (including empty and one-token sequences), group sizes, block
sizes that do and do not divide the 64-key tile, top-k from 1 to more than the
number of blocks; bf16 and fp32 forward, decode with and without the
caller's block means.  Every row and every gradient element is compared with the
oracle under the tolerances of tests/parity.py; a decode row with near-tied
gate scores is compared over the admissible selection closest to it, as in
tests/test_gpu_decode.py.
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


def random_case(seed, max_tokens, nonempty=False):
    rng = np.random.default_rng(seed)
    S = int(rng.integers(1, 5))
    lens = []
    for _ in range(S):
        r = rng.random()
        if r < 0.15 and not nonempty:
            lens.append(0)
        elif r < 0.3:
            lens.append(int(rng.integers(1, 8)))
        else:
            lens.append(int(rng.integers(8, max_tokens)))
    if sum(lens) == 0:
        lens[0] = int(rng.integers(8, max_tokens))
    hkv = int(rng.choice([1, 2, 4]))
    G = int(rng.choice([1, 2, 3, 4, 8]))
    B = int(rng.choice([1, 5, 16, 48, 64, 100, 128, 200, 256]))
    topk = int(rng.integers(1, 9))
    return tuple(lens), G * hkv, hkv, B, topk


FWD_SEEDS = list(range(100, 124))
BWD_SEEDS = list(range(200, 212))
DEC_SEEDS = list(range(300, 312))
F32_SEEDS = list(range(400, 408))


@pytest.mark.parametrize("seed", FWD_SEEDS)
def test_random_forward(seed):
    seqlens, hq, hkv, B, topk = random_case(seed, 700)
    q, k, v, cu = inputs.make(seqlens, hq, hkv, 128, torch.bfloat16, B, 0.5, seed, device=DEV)
    r = parity.moba_parity(q, k, v, cu, B, topk, dtype="bf16")
    print(seqlens, hq, hkv, B, topk, "max %.2e mean %.2e lse %.2e ties %d" %
          (r["max_abs"], r["mean_abs"], r["lse_max_abs"], r["tie_rows"]))


@pytest.mark.parametrize("seed", F32_SEEDS)
def test_random_forward_f32(seed):
    """fp32 inputs: the selection must equal the oracle's exactly."""
    seqlens, hq, hkv, B, topk = random_case(seed, 600)
    q, k, v, cu = inputs.make(seqlens, hq, hkv, 128, torch.float32, B, 0.5, seed, device=DEV)
    r = parity.moba_parity(q, k, v, cu, B, topk, dtype="f32")
    print(seqlens, hq, hkv, B, topk, "max %.2e lse %.2e" % (r["max_abs"], r["lse_max_abs"]))


@pytest.mark.parametrize("seed", BWD_SEEDS)
def test_random_backward(seed):
    seqlens, hq, hkv, B, topk = random_case(seed, 400)
    q, k, v, cu = inputs.make(seqlens, hq, hkv, 128, torch.bfloat16, B, 0.5, seed, device=DEV)
    dout = inputs.make_dout(q.shape, q.dtype, seed, device=DEV)
    res = parity.moba_backward_parity(q, k, v, cu, B, topk, dout)
    print(seqlens, hq, hkv, B, topk, res)


@pytest.mark.parametrize("seed", DEC_SEEDS)
@pytest.mark.parametrize("mode", ["moba", "moba_kbar", "full"])
def test_random_decode(seed, mode):
    seqlens, hq, hkv, B, topk = random_case(seed, 900, nonempty=True)
    q, k, v, cu = inputs.make(seqlens, hq, hkv, 128, torch.bfloat16, B, 0.5, seed, device=DEV)
    T, S = q.shape[0], len(seqlens)
    last = (cu[1:] - 1).to(torch.int64)
    qd = q[last.to(DEV)].contiguous()
    kbar = binding.pool(k, cu, B) if mode == "moba_kbar" else None
    out, lse = binding.decode(qd, k, v, cu, B, 0 if mode == "full" else topk, kbar=kbar)
    torch.cuda.synchronize()
    rows = np.array([int(t) * hq + h for t in last for h in range(hq)], np.int64)
    q_rows = inputs.to_oracle(qd.reshape(S * hq, 128))
    kn, vn, cun = inputs.to_oracle(k), inputs.to_oracle(v), cu.numpy()
    gout = out.float().cpu().numpy().reshape(S * hq, 128)
    glse = lse.cpu().numpy().T.reshape(S * hq)
    if mode == "full":
        sel = np.zeros((len(rows), 1), np.int32)
        oout, olse = oracle.attend_rows(q_rows, T, hq, kn, vn, cun, max(seqlens), sel, rows)
        mx, mean, lmx = parity.compare_outputs(gout, glse, oout, olse, "bf16", mode)
        multi = 0
    else:
        mx, mean, lmx, multi, _ = parity.check_rows_any_selection(gout, glse, q_rows, rows, T, hq,
                                                                  kn, vn, cun, B, topk, mode)
    print(seqlens, hq, hkv, B, topk, mode, "near-tie rows %d max %.2e" % (multi, mx))
