"""Parity of the HIP backward (moba_backward) with the oracle's fp64
gradients, through the C ABI.

The cases span several dQ tiles and dK/dV key tiles and row chunks, ragged
sequence tails, empty sequences, block sizes that do and do not divide the
64-key tile or the 256-key dK/dV tile, GQA groups up to 8, top-1 (no routed
rows) and top-k beyond the number of blocks (dense causal).
"""
import numpy as np
import pytest
import torch

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
    ((1000, 0, 517), 4, 2, 128, 3),
    ((777,), 8, 2, 100, 4),
    ((513, 129, 64), 4, 1, 48, 5),
    ((640,), 3, 3, 64, 1),
    ((700,), 4, 4, 96, 20),
    ((2048,), 16, 2, 256, 3),
    ((333, 1), 2, 1, 7, 6),
    ((1500,), 4, 1, 512, 3),
    ((1300, 900), 8, 1, 300, 3),
    ((40, 17), 2, 1, 1, 4),      # one-key blocks
    ((600, 45), 16, 1, 64, 3),   # 16 query heads per kv-head
    ((200, 37), 64, 1, 32, 4),   # 64 query heads per kv-head
    ((1500, 300), 4, 2, 16, 24),  # 23 history slots: long row lists per 16-key block
    ((1000, 0, 333), 8, 2, 8, 32),  # 31 history slots over up to 124 blocks
]


@pytest.mark.parametrize("seqlens,hq,hkv,B,topk", CASES,
                         ids=["-".join(map(str, c[0])) + "_h%dx%d_B%d_k%d" % c[1:] for c in CASES])
def test_backward_small(seqlens, hq, hkv, B, topk):
    seed = sum(seqlens) + B + 1
    print("case", seqlens, hq, hkv, B, topk, flush=True)
    q, k, v, cu = inputs.make(seqlens, hq, hkv, 128, torch.bfloat16, B, 0.5, seed, device=DEV)
    dout = inputs.make_dout(q.shape, torch.bfloat16, seed, device=DEV)
    r = parity.moba_backward_parity(q, k, v, cu, B, topk, dout)
    print("tie_rows %d  dq %.2e/%.2e  dk %.2e/%.2e  dv %.2e/%.2e (max |err|/(|ref|+c), "
          "mean |err|/mean |ref|)" % (r["tie_rows"], *r["dq"], *r["dk"], *r["dv"]), flush=True)


def test_backward_is_deterministic():
    q, k, v, cu = inputs.make((1500, 700), 8, 2, 128, torch.bfloat16, 256, 0.5, 5, device=DEV)
    dout = inputs.make_dout(q.shape, torch.bfloat16, 5, device=DEV)
    out, lse = binding.forward(q, k, v, cu, 256, 3)
    a = binding.backward(q, k, v, cu, 256, 3, out, lse, dout)
    b = binding.backward(q, k, v, cu, 256, 3, out, lse, dout)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_backward_rejects_f32():
    q, k, v, cu = inputs.make((100,), 2, 2, 128, torch.float32, 32, 0.0, 1, device=DEV)
    out, lse = binding.forward(q, k, v, cu, 32, 2)
    with pytest.raises(binding.MobaError) as e:
        binding.backward(q, k, v, cu, 32, 2, out, lse, torch.zeros_like(q))
    assert e.value.name == "MOBA_ERR_DTYPE"


DENSE = [((300,), 2, 2), ((1000, 0, 517), 4, 2), ((129, 64, 1), 8, 1), ((1300,), 4, 1)]


@pytest.mark.parametrize("seqlens,hq,hkv", DENSE,
                         ids=["-".join(map(str, c[0])) + "_h%dx%d" % c[1:] for c in DENSE])
def test_dense_backward(seqlens, hq, hkv):
    """moba_dense_backward: gradients of causal full attention (Eq. 1), the
    full-attention side of the per-call switch, against the oracle's gradients
    for one block per sequence (every row attends its whole causal prefix)."""
    from oracle import oracle

    seed = sum(seqlens) + 11
    q, k, v, cu = inputs.make(seqlens, hq, hkv, 128, torch.bfloat16, 64, 0.5, seed, device=DEV)
    dout = inputs.make_dout(q.shape, torch.bfloat16, seed, device=DEV)
    out, lse = binding.dense_forward(q, k, v, cu)
    dq, dk, dv = binding.dense_backward(q, k, v, cu, out, lse, dout)
    torch.cuda.synchronize()
    T = q.shape[0]
    B = max(max(seqlens), 1)
    sel = np.zeros((T * hq, 1), np.int32)
    qn, kn, vn = parity.host_inputs(q, k, v)
    odq, odk, odv, cq, ck, cv = oracle.attend_backward(qn, kn, vn, inputs.to_oracle(dout),
                                                       cu.numpy(), B, sel, kv_window="all",
                                                       with_bounds=True)
    for name, g, ref, c in (("dq", dq, odq, cq), ("dk", dk, odk, ck), ("dv", dv, odv, cv)):
        g = g.float().cpu().numpy().astype(np.float64).reshape(ref.shape)
        err = np.abs(g - ref)
        ratio = float((err / (np.abs(ref) + c + 1e-30)).max())
        mean_rel = float(err.mean() / np.abs(ref).mean())
        print("%s: %.2e of (|ref| + c), mean %.2e" % (name, ratio, mean_rel))
        assert ratio <= parity.BWD_ELEM_U and mean_rel <= parity.BWD_MEAN_REL, name


def test_wait_give_up_is_reported(monkeypatch):
    """The dK/dV kernel's bounded hand-over wait, forced from the host to
    give up on every subtile (every kernel still runs to its end): the
    give-ups are counted and reported, as MOBA_ERR_HIP under MOBA_DEBUG_SYNC;
    a normal call afterwards counts none and is correct again."""
    q, k, v, cu = inputs.make((700, 300), 4, 2, 128, torch.bfloat16, 128, 0.5, 91, device=DEV)
    out, lse = binding.forward(q, k, v, cu, 128, 3)
    dout = inputs.make_dout(q.shape, torch.bfloat16, 91, device=DEV)
    ref = binding.backward(q, k, v, cu, 128, 3, out, lse, dout)
    assert binding.take_wait_timeouts() == 0
    monkeypatch.setenv("MOBA_FORCE_WAIT_TIMEOUT", "1")
    binding.backward(q, k, v, cu, 128, 3, out, lse, dout)
    assert binding.take_wait_timeouts() > 0
    monkeypatch.setenv("MOBA_DEBUG_SYNC", "1")
    with pytest.raises(binding.MobaError) as e:
        binding.backward(q, k, v, cu, 128, 3, out, lse, dout)
    assert e.value.name == "MOBA_ERR_HIP"
    monkeypatch.delenv("MOBA_FORCE_WAIT_TIMEOUT")
    again = binding.backward(q, k, v, cu, 128, 3, out, lse, dout)
    monkeypatch.delenv("MOBA_DEBUG_SYNC")
    assert binding.take_wait_timeouts() == 0
    for x, y in zip(ref, again):
        assert torch.equal(x, y)
