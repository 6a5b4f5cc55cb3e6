"""moba_decode_noalloc (the decode entry point that allocates nothing; its
buffers live in a static device array) against moba_decode, through the C
ABI: on the same inputs the two run the same kernels and must give
bit-identical outputs, over two calls in a row (the second with a smaller
problem, so the array holds the first call's contents when the second
starts); MoBA mode with and without the caller's block means, and full
attention.  Sizes beyond the array and device offsets are refused before any
work is enqueued."""
import numpy as np
import pytest
import torch

from paper_2502_13189_amd import binding, inputs

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.load()


def decode_inputs(seqlens, hq, hkv, B, seed):
    q, k, v, cu = inputs.make(seqlens, hq, hkv, 128, torch.bfloat16, B, 0.5, seed, device=DEV)
    last = (cu[1:] - 1).to(torch.int64).to(DEV)
    return q[last].contiguous(), k, v, cu


def both(qd, k, v, cu, B, topk, kbar):
    o1, l1 = binding.decode(qd, k, v, cu, B, topk, kbar=kbar)
    o2 = torch.full_like(qd, float("nan"))
    l2 = torch.full((qd.shape[1], qd.shape[0]), float("nan"), device=DEV)
    binding.decode_noalloc(qd, k, v, cu, B, topk, o2, l2, kbar=kbar)
    torch.cuda.synchronize()
    return o1, l1, o2, l2


@pytest.mark.parametrize("mode", ["moba_kbar", "moba", "full"])
def test_noalloc_decode_equals_decode_twice(mode):
    cases = [((24000, 300, 4097), 16, 2, 4096, 5, 11),   # two combine shares per row
             ((700, 129), 4, 1, 64, 3, 12)]                # the smaller second call
    for seqlens, hq, hkv, B, topk, seed in cases:
        qd, k, v, cu = decode_inputs(seqlens, hq, hkv, B, seed)
        kbar = binding.pool(k, cu, B) if mode == "moba_kbar" else None
        kk = 0 if mode == "full" else topk
        o1, l1, o2, l2 = both(qd, k, v, cu, B, kk, kbar)
        assert torch.equal(o1, o2), (mode, seqlens)
        assert torch.equal(l1, l2), (mode, seqlens)
        print(mode, seqlens, "bit-identical")


def test_noalloc_decode_refuses_what_it_cannot_hold():
    # full attention over 16 sequences of 128K tokens with 32 query heads
    # needs 512 rows x 512 partials x 516 bytes, above the array's size
    seqlens, hq, hkv = (131072,) * 16, 32, 8
    T = sum(seqlens)
    k = torch.zeros((T, hkv, 128), dtype=torch.bfloat16, device=DEV)
    qd = torch.zeros((len(seqlens), hq, 128), dtype=torch.bfloat16, device=DEV)
    cu = inputs.cu_seqlens(seqlens)
    o = torch.zeros_like(qd)
    l = torch.zeros((hq, len(seqlens)), device=DEV)
    with pytest.raises(binding.MobaError) as e:
        binding.decode_noalloc(qd, k, k, cu, 4096, 0, o, l)
    assert e.value.name == "MOBA_ERR_NO_MEMORY"
    assert bool((o == 0).all()) and bool((l == 0).all())
    # device offsets would need a device-to-host copy through pinned memory
    with pytest.raises(binding.MobaError) as e:
        binding.decode_noalloc(qd[:1], k[:1000], k[:1000], torch.tensor([0, 1000], dtype=torch.int32,
                                                                       device=DEV), 64, 3, o[:1],
                               l[:, :1].contiguous())
    assert e.value.name == "MOBA_ERR_UNSUPPORTED"
