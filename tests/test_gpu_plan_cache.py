"""The per-shape tables (sequence offsets, tile lists) are built on the host
and copied on the caller's stream without synchronizing the device, into a
few cached slots.  These tests enqueue calls with more distinct cu_seqlens
than there are slots, with no synchronization between them, so that tables
are rebuilt while earlier calls' kernels are still queued, and require the
results to equal, bit for bit, those of the same calls made one at a time
with a synchronization after each (every kernel here is deterministic).
"""
import pytest
import torch

from paper_2502_13189_amd import binding, inputs

pytestmark = pytest.mark.gpu
DEV = "cuda:0"

# six partitions of 3000 tokens: more than the slots the library keeps
SPLITS = [(3000,), (1000, 2000), (1500, 1500), (10, 2990), (700, 700, 1600), (2999, 1)]


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.load()


def _data(T, hq, hkv, seed):
    q, k, v, _ = inputs.make((T,), hq, hkv, 128, torch.bfloat16, 64, 0.5, seed, device=DEV)
    return q, k, v


def test_forward_backward_with_tables_rebuilt_in_flight():
    q, k, v = _data(3000, 4, 2, 11)
    dout = inputs.make_dout(q.shape, q.dtype, 11, device=DEV)
    cus = [inputs.cu_seqlens(s) for s in SPLITS]
    ref = []
    for cu in cus:
        o, l = binding.forward(q, k, v, cu, 64, 3)
        g = binding.backward(q, k, v, cu, 64, 3, o, l, dout)
        torch.cuda.synchronize()
        ref.append((o.clone(), l.clone()) + tuple(x.clone() for x in g))
    for rep in range(2):
        got = []
        for cu in cus:  # no synchronization inside the loop
            o, l = binding.forward(q, k, v, cu, 64, 3)
            got.append((o, l) + tuple(binding.backward(q, k, v, cu, 64, 3, o, l, dout)))
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(got, ref)):
            for name, x, y in zip(("out", "lse", "dq", "dk", "dv"), a, b):
                assert torch.equal(x, y), "split %s, %s differs (pass %d)" % (SPLITS[i], name, rep)


def test_moba_and_dense_interleaved():
    q, k, v = _data(3000, 8, 2, 12)
    cus = [inputs.cu_seqlens(s) for s in SPLITS]
    ref = []
    for cu in cus:
        m = binding.forward(q, k, v, cu, 64, 3)
        d = binding.dense_forward(q, k, v, cu)
        torch.cuda.synchronize()
        ref.append(tuple(x.clone() for x in m + d))
    got = [binding.forward(q, k, v, cu, 64, 3) + binding.dense_forward(q, k, v, cu) for cu in cus]
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(zip(got, ref)):
        for x, y in zip(a, b):
            assert torch.equal(x, y), "split %s differs" % (SPLITS[i],)


@pytest.mark.parametrize("topk", [3, 0])
def test_decode_growing_cache(topk):
    """A decode loop over a growing two-sequence cache: new cu_seqlens every
    step (the second sequence grows; the first is fixed)."""
    L0, L1, steps, hq, hkv, B = 700, 300, 40, 8, 2, 64
    g = torch.Generator(device=DEV).manual_seed(13)
    k = torch.randn((L0 + L1 + steps, hkv, 128), device=DEV, generator=g).to(torch.bfloat16)
    v = torch.randn((L0 + L1 + steps, hkv, 128), device=DEV, generator=g).to(torch.bfloat16)
    qd = torch.randn((steps, 2, hq, 128), device=DEV, generator=g).to(torch.bfloat16)
    cus = [torch.tensor([0, L0, L0 + L1 + i + 1], dtype=torch.int32) for i in range(steps)]
    ref = []
    for i, cu in enumerate(cus):
        T = int(cu[-1])
        o, l = binding.decode(qd[i], k[:T], v[:T], cu, B, topk)
        torch.cuda.synchronize()
        ref.append((o.clone(), l.clone()))
    got = []
    for i, cu in enumerate(cus):
        T = int(cu[-1])
        got.append(binding.decode(qd[i], k[:T], v[:T], cu, B, topk))
    torch.cuda.synchronize()
    for i, ((o, l), (ro, rl)) in enumerate(zip(got, ref)):
        assert torch.equal(o, ro) and torch.equal(l, rl), "step %d differs" % i


def test_calls_on_a_side_stream():
    """New shapes first seen on a side stream (default priority): their
    tables are copied on that stream.  The streams are ordered with events,
    as calls on different streams must not overlap."""
    q, k, v = _data(3000, 4, 2, 21)
    dout = inputs.make_dout(q.shape, q.dtype, 21, device=DEV)
    splits = [(1234, 1766), (64, 2936), (3000,)]
    cus = [inputs.cu_seqlens(s) for s in splits]
    ref = []
    for cu in cus:
        o, l = binding.forward(q, k, v, cu, 64, 3)
        g = binding.backward(q, k, v, cu, 64, 3, o, l, dout)
        torch.cuda.synchronize()
        ref.append((o.clone(), l.clone()) + tuple(x.clone() for x in g))
    binding.release_workspace()  # drops the cached tables too
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream(device=DEV)
    got = []
    for i, cu in enumerate(cus):
        st = side if i % 2 == 0 else main
        st.wait_stream(main if st is side else side)
        with torch.cuda.stream(st):
            o, l = binding.forward(q, k, v, cu, 64, 3)
            got.append((o, l) + tuple(binding.backward(q, k, v, cu, 64, 3, o, l, dout)))
    main.wait_stream(side)
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(zip(got, ref)):
        for name, x, y in zip(("out", "lse", "dq", "dk", "dv"), a, b):
            assert torch.equal(x, y), "split %s, %s differs" % (splits[i], name)
