"""Parity of the HIP library with the fp64 oracle, through the C ABI.

Small cases cover every row; they span several attention tiles, ragged
sequence tails, empty sequences, block sizes that do and do not divide the
64-key tile, GQA groups, fp32 and bf16.  The full-size workloads compare every
row where the oracle finishes in seconds and a fixed row sample otherwise.
"""
import os

import numpy as np
import pytest
import torch

from paper_2502_13189_amd import binding, inputs
from oracle import oracle
import parity

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _gpu_available():
    return torch.cuda.is_available()


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not _gpu_available():
        pytest.skip("no GPU")
    binding.load()


def make(seqlens, hq, hkv, dtype, B, offset=0.0, seed=0):
    q, k, v, cu = inputs.make(seqlens, hq, hkv, 128, dtype, B, offset, seed, device=DEV)
    return q, k, v, cu


SMALL = [
    # seqlens, hq, hkv, B, topk, dtype
    ((300,), 2, 2, 64, 3, torch.bfloat16),
    ((1000, 0, 517), 4, 2, 128, 3, torch.bfloat16),
    ((777,), 8, 2, 100, 4, torch.bfloat16),
    ((513, 129, 64), 4, 1, 48, 5, torch.bfloat16),
    ((640,), 3, 3, 64, 1, torch.bfloat16),
    ((700,), 4, 4, 96, 20, torch.bfloat16),
    ((2048,), 16, 2, 256, 3, torch.bfloat16),
    ((333, 1), 2, 1, 7, 6, torch.bfloat16),
    ((40, 17), 2, 1, 1, 4, torch.bfloat16),        # one-key blocks
    ((600,), 32, 1, 64, 3, torch.bfloat16),        # 32 query heads per kv-head
    ((300, 45), 128, 1, 64, 3, torch.bfloat16),    # the largest group, 128 query heads per kv-head
    ((257, 3), 4, 2, 4096, 2, torch.bfloat16),     # block larger than every sequence
    ((4000,), 2, 1, 1, 3, torch.bfloat16),         # 4000 blocks: routing ranks without its LDS prefix table
    # more than one 32-block gate chunk, for each list size the gate bounds
    # from below (k-1 = 1, 11, 15) before inserting
    ((1500,), 4, 4, 16, 2, torch.bfloat16),
    ((3000, 70), 4, 2, 16, 12, torch.bfloat16),
    ((2500,), 2, 1, 8, 16, torch.bfloat16),
    ((1500, 300), 4, 2, 16, 40, torch.bfloat16),  # k-1 = 39: the 63-place gate list, entries routed one by one
    ((1500, 300), 4, 2, 16, 24, torch.bfloat16),  # k-1 = 23 in the 31-place list (8 places blocked)
    ((1000, 0, 333), 8, 2, 8, 32, torch.bfloat16),  # k-1 = 31 fills the 31-place list, up to 124 blocks
    ((900, 77), 2, 1, 16, 24, torch.float32),       # fp32 gate, 31-place list: selection bit-exact
    ((300,), 2, 2, 64, 3, torch.float32),
    ((600, 250), 4, 2, 128, 4, torch.float32),
    ((515,), 2, 1, 50, 3, torch.float32),
]


@pytest.mark.parametrize("seqlens,hq,hkv,B,topk,dtype", SMALL,
                         ids=["-".join(map(str, c[0])) + "_h%dx%d_B%d_k%d_%s" % (c[1], c[2], c[3], c[4], str(c[5])[6:]) for c in SMALL])
def test_moba_small(seqlens, hq, hkv, B, topk, dtype):
    q, k, v, cu = make(seqlens, hq, hkv, dtype, B, offset=0.5, seed=sum(seqlens) + B)
    r = parity.moba_parity(q, k, v, cu, B, topk, dtype="f32" if dtype == torch.float32 else "bf16")
    print("rows %d tie_rows %d max_abs %.2e mean_abs %.2e lse %.2e" %
          (r["rows"], r["tie_rows"], r["max_abs"], r["mean_abs"], r["lse_max_abs"]))


@pytest.mark.parametrize("seqlens,hq,hkv,dtype", [
    ((300,), 2, 2, torch.bfloat16), ((1000, 0, 517), 4, 2, torch.bfloat16),
    ((129, 64, 1), 8, 1, torch.bfloat16), ((300, 77), 2, 1, torch.float32)])
def test_dense_small(seqlens, hq, hkv, dtype):
    q, k, v, cu = make(seqlens, hq, hkv, dtype, 64, seed=7)
    parity.dense_parity(q, k, v, cu, dtype="f32" if dtype == torch.float32 else "bf16")


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_pool_matches_oracle(dtype):
    seqlens, B = (1000, 0, 333, 64), 100
    q, k, v, cu = make(seqlens, 4, 2, dtype, B, offset=0.5, seed=3)
    kbar = binding.pool(k, cu, B).cpu().numpy().astype(np.float64)
    ref, kabs = oracle.pool(inputs.to_oracle(k), cu.numpy(), B, with_abs=True)
    # fp64 accumulation rounded once to fp32: within one fp32 ulp of the mean
    tol = 2.0 ** -23 * np.abs(ref) + 1e-12 * kabs
    assert np.all(np.abs(kbar - ref) <= tol)


@pytest.mark.parametrize("B,L,topk", [(64, 900, 4), (16, 900, 4), (8, 1200, 12), (4, 1000, 16),
                                      (4, 1000, 32)])
def test_select_constructed_ties(B, L, topk):
    """Every block holds the same keys: all scores tie exactly and the lower
    block index must win on the GPU too (also where rows have more than one
    32-block gate chunk and the gate first bounds the list from below)."""
    q, k, v, cu = make((L,), 4, 2, torch.bfloat16, B, seed=5)
    blk = k[:B].clone()
    k = blk.repeat((L + B - 1) // B, 1, 1)[:L].contiguous()
    sel = binding.select(q, k, cu, B, topk).cpu().numpy()
    for t in range(L):
        c = t // B
        expect = list(range(min(topk - 1, c))) + [c] + [-1] * (topk - 1 - min(topk - 1, c))
        assert (sel[t] == np.array(expect)).all(), (t, sel[t], expect)


def test_select_scores_within_bound():
    """The GPU's fp32 gate scores stay within the tie tolerance of the fp64
    scores (this is what justifies the tie-aware comparison)."""
    seqlens, B, topk = (2000, 900), 128, 3
    q, k, v, cu = make(seqlens, 4, 2, torch.bfloat16, B, offset=0.5, seed=9)
    nmax = 16
    sel, sc = binding.select(q, k, cu, B, topk, nmax=nmax)
    qn, kn = inputs.to_oracle(q), inputs.to_oracle(k)
    kbar, kabs = oracle.pool(kn, cu.numpy(), B, with_abs=True)
    rows = np.arange(q.shape[0] * q.shape[1])
    _, osc = oracle.select(qn, kbar, cu.numpy(), B, topk, rows=rows, nmax=nmax)
    gsc = sc.view(-1, nmax).cpu().numpy().astype(np.float64)
    valid = ~np.isnan(osc)
    assert np.array_equal(valid, ~np.isnan(gsc))
    T, Hq = q.shape[0], q.shape[1]
    qa = np.abs(parity._widen(qn)).reshape(T * Hq, 128)
    boff = parity.block_offsets(cu.numpy(), B)
    s_of = parity.seq_of_tokens(cu.numpy(), rows // Hq)
    g_of = (rows % Hq) // (Hq // 2)
    for j in range(nmax):
        m = valid[:, j]
        if not m.any():
            continue
        a = kabs[np.array(boff)[s_of[m]] + j, g_of[m]]
        tau = parity.TAU_SCALE * np.einsum("rd,rd->r", qa[m], a)
        assert np.all(np.abs(gsc[m, j] - osc[m, j]) <= tau)


ROUTE_CASES = [
    # seqlens, hq, hkv, B, topk
    ((1500, 0, 700, 33), 8, 2, 64, 4),
    ((9000, 0, 3000), 8, 2, 128, 12),  # several routing chunks per sequence, LDS-staged runs
    ((2000, 1000), 6, 2, 32, 5),       # groups of 3 query heads: rounds of 255 rows
    ((700,), 2, 1, 1, 64),             # 700 one-key blocks, 63 per row: entries written directly
]


def _cpu_route(sel_h, cun, T, hq, hkv, B, topk):
    """The bins of Algorithm 1's index_select step, by direct enumeration:
    for every row, in row order, its history slots x < min(topk - 1, c);
    a slot holding a block outside [0, c) is not routed."""
    G = hq // hkv
    boff = parity.block_offsets(cun, B)
    nb = oracle.num_blocks(cun, B)
    bins = [[] for _ in range(hkv * nb)]
    for t in range(T):
        s = int(parity.seq_of_tokens(cun, t))
        c = (t - cun[s]) // B
        for h in range(hq):
            g, hl = h // G, h % G
            r = g * T * G + t * G + hl
            for x in range(min(topk - 1, c)):
                j = int(sel_h[t, h, x])
                if 0 <= j < c:
                    bins[g * nb + boff[s] + j].append(r * (topk - 1) + x)
    counts = np.array([len(b) for b in bins])
    offsets = np.concatenate([[0], np.cumsum(counts)])
    entries = np.array([e for b in bins for e in b], dtype=np.int64)
    return counts, offsets, entries


def _check_route(sel, cu, T, hq, hkv, B, topk):
    counts, offsets, entries = binding.route(sel, cu, B, hkv)
    exp_counts, exp_off, exp_entries = _cpu_route(sel.cpu().numpy(), cu.numpy(), T, hq, hkv,
                                                  B, topk)
    assert np.array_equal(counts.cpu().numpy(), exp_counts)
    assert np.array_equal(offsets.cpu().numpy(), exp_off)
    n = int(exp_off[-1])
    assert np.array_equal(entries[:n].cpu().numpy().astype(np.int64) & 0xffffffff, exp_entries)


@pytest.mark.parametrize("seqlens,hq,hkv,B,topk", ROUTE_CASES,
                         ids=["-".join(map(str, c[0])) + "_h%dx%d_B%d_k%d" % c[1:]
                              for c in ROUTE_CASES])
def test_route_matches_cpu_inversion(seqlens, hq, hkv, B, topk):
    """Algorithm 1's index_select step: every bin's list holds exactly the
    history selections of its (kv-head, block), in row order."""
    q, k, v, cu = make(seqlens, hq, hkv, torch.bfloat16, B, offset=0.5, seed=11)
    sel = binding.select(q, k, cu, B, topk)
    _check_route(sel, cu, q.shape[0], hq, hkv, B, topk)


ROUTE_BAD_CASES = [ROUTE_CASES[i] for i in (1, 2, 3)]


@pytest.mark.parametrize("seqlens,hq,hkv,B,topk", ROUTE_BAD_CASES,
                         ids=["-".join(map(str, c[0])) + "_h%dx%d_B%d_k%d" % c[1:]
                              for c in ROUTE_BAD_CASES])
def test_route_skips_out_of_range_slots(seqlens, hq, hkv, B, topk):
    """A history slot of a caller's sel that holds no past block (negative,
    the current block or later) is skipped alike by the count and the scatter,
    so the bins hold exactly the in-range selections."""
    q, k, v, cu = make(seqlens, hq, hkv, torch.bfloat16, B, offset=0.5, seed=12)
    sel = binding.select(q, k, cu, B, topk)
    T = q.shape[0]
    cun = cu.numpy()
    rng = np.random.default_rng(5)
    sel_h = sel.cpu().numpy().copy()
    bad = [-1, -(2 ** 31), 0, 5, 10 ** 6]  # 0 and 5 become c + 0 and c + 5
    planted = 0
    for t in rng.choice(T, size=min(T, 400), replace=False):
        s = int(parity.seq_of_tokens(cun, t))
        c = (int(t) - cun[s]) // B
        if min(topk - 1, c) == 0:
            continue
        h = int(rng.integers(hq))
        x = int(rng.integers(min(topk - 1, c)))
        v_ = bad[planted % len(bad)]
        sel_h[t, h, x] = c + v_ if v_ in (0, 5) else v_
        planted += 1
    assert planted > 50
    _check_route(torch.from_numpy(sel_h).to(sel.device), cu, T, hq, hkv, B, topk)


def test_deterministic():
    q, k, v, cu = make((1500, 800), 8, 2, torch.bfloat16, 128, offset=0.5, seed=13)
    o1, l1 = binding.forward(q, k, v, cu, 128, 4)
    o2, l2 = binding.forward(q, k, v, cu, 128, 4)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_gqa_equals_mha_with_repeated_kv():
    q, k, v, cu = make((900, 300), 8, 2, torch.bfloat16, 64, offset=0.5, seed=17)
    o1, l1 = binding.forward(q, k, v, cu, 64, 3)
    o2, l2 = binding.forward(q, k.repeat_interleave(4, dim=1).contiguous(),
                             v.repeat_interleave(4, dim=1).contiguous(), cu, 64, 3)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_varlen_equals_separate_calls():
    seqlens = (700, 0, 1200, 65)
    q, k, v, cu = make(seqlens, 4, 2, torch.bfloat16, 128, offset=0.5, seed=19)
    o, l = binding.forward(q, k, v, cu, 128, 3)
    a = 0
    for L in seqlens:
        if L == 0:
            continue
        cs = torch.tensor([0, L], dtype=torch.int32)
        os_, ls = binding.forward(q[a:a + L].contiguous(), k[a:a + L].contiguous(),
                                  v[a:a + L].contiguous(), cs, 128, 3)
        assert torch.equal(os_, o[a:a + L]) and torch.equal(ls, l[:, a:a + L])
        a += L


def test_strided_inputs():
    """q, k, v as column slices of one packed projection (token stride > H*D)."""
    T, hq, hkv = 1100, 4, 2
    q, k, v, cu = make((T,), hq, hkv, torch.bfloat16, 128, offset=0.5, seed=23)
    packed = torch.cat([q, k, v], dim=1)
    qs, ks, vs = packed[:, :hq], packed[:, hq:hq + hkv], packed[:, hq + hkv:]
    o1, l1 = binding.forward(q, k, v, cu, 128, 3)
    o2, l2 = binding.forward(qs, ks, vs, cu, 128, 3)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_workspace_chunking_is_invisible(monkeypatch):
    """A small workspace cap splits the attention into kv-head chunks; the
    result must not change."""
    q, k, v, cu = make((2000, 900), 8, 4, torch.bfloat16, 128, offset=0.5, seed=29)
    o1, l1 = binding.forward(q, k, v, cu, 128, 4)
    torch.cuda.synchronize()
    monkeypatch.setenv("MOBA_WORKSPACE_LIMIT_BYTES", str(40 << 20))
    o2, l2 = binding.forward(q, k, v, cu, 128, 4)
    torch.cuda.synchronize()
    monkeypatch.setenv("MOBA_WORKSPACE_LIMIT_BYTES", str(1 << 20))
    with pytest.raises(binding.MobaError) as ei:
        binding.forward(q, k, v, cu, 128, 4)
    assert ei.value.name == "MOBA_ERR_NO_MEMORY"
    monkeypatch.delenv("MOBA_WORKSPACE_LIMIT_BYTES")
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_chunked_attention_matches_one_pass(monkeypatch):
    """Caps below the one-pass workspace (moba_workspace_bytes) split the
    attention into 2 to 8 chunks of kv-heads that reuse one partial buffer;
    every split must give the one-pass result bit for bit (the merge count
    shows the chunk count)."""
    seqlens, hq, hkv, B, topk = (2100, 0, 1300), 16, 8, 64, 5
    q, k, v, cu = make(seqlens, hq, hkv, torch.bfloat16, B, offset=0.5, seed=33)
    nblk, _ = binding.route_size(cu, B, topk, hq)
    one = binding.workspace_bytes(q.shape[0], hq, hkv, nblk, topk)
    o1, l1 = binding.forward(q, k, v, cu, B, topk)
    torch.cuda.synchronize()
    chunks = []
    for frac in (1.0, 0.5, 0.4, 0.3, 0.25, 0.2, 0.15, 0.12):
        monkeypatch.setenv("MOBA_WORKSPACE_LIMIT_BYTES", str(int(one * frac)))
        binding.profile_read()
        binding.profile_enable(True)
        try:
            o2, l2 = binding.forward(q, k, v, cu, B, topk)
        except binding.MobaError as e:  # below the fixed part plus one kv-head
            binding.profile_enable(False)
            assert e.name == "MOBA_ERR_NO_MEMORY"
            continue
        torch.cuda.synchronize()
        binding.profile_enable(False)
        chunks.append(binding.profile_read().get("merge", (0, 0.0))[0])
        assert torch.equal(o1, o2) and torch.equal(l1, l2), frac
    monkeypatch.delenv("MOBA_WORKSPACE_LIMIT_BYTES")
    print("merge launches per cap:", chunks)
    assert len(chunks) >= 3 and chunks[0] == 1 and max(chunks) >= 4, chunks


def test_device_cu_seqlens():
    q, k, v, cu = make((500, 300), 4, 2, torch.bfloat16, 64, seed=31)
    o1, l1 = binding.forward(q, k, v, cu, 64, 3)
    o2, l2 = binding.forward(q, k, v, cu.to(DEV), 64, 3)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_device_cu_seqlens_written_on_a_side_stream():
    """A device cu_seqlens written by work on the caller's (non-default)
    stream is read after that work: the library copies it on that stream.
    The offsets are first set to another valid batch, then overwritten on the
    side stream behind a long matrix product, and the call is made on the
    side stream without any host synchronization in between."""
    q, k, v, cu = make((500, 300), 4, 2, torch.bfloat16, 64, seed=31)
    o1, l1 = binding.forward(q, k, v, cu, 64, 3)
    decoy = torch.tensor([0, 100, 800], dtype=torch.int32, device=DEV)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        a = torch.randn(8192, 8192, device=DEV)
        for _ in range(4):
            a = a @ a * 1e-4
        decoy.copy_(cu.to(DEV, non_blocking=True) + (a[0, 0] * 0).to(torch.int32))
        o2, l2 = binding.forward(q, k, v, decoy, 64, 3, stream=side)
    side.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_workspace_bytes_is_enough_for_one_pass(monkeypatch):
    """With the workspace cap at moba_workspace_bytes' figure the forward
    runs its history attention in one pass (one launch per call), and the
    workspace it holds is within the figure."""
    seqlens, hq, hkv, B, topk = (3000, 0, 1700), 8, 2, 128, 4
    q, k, v, cu = make(seqlens, hq, hkv, torch.bfloat16, B, seed=43)
    nb, _ = binding.route_size(cu, B, topk, hq)
    need = binding.workspace_bytes(q.shape[0], hq, hkv, nb, topk)
    binding.release_workspace()
    monkeypatch.setenv("MOBA_WORKSPACE_LIMIT_BYTES", str(need))
    binding.profile_enable(True)
    binding.profile_read()
    o1, l1 = binding.forward(q, k, v, cu, B, topk)
    ph = binding.profile_read()
    binding.profile_enable(False)
    monkeypatch.delenv("MOBA_WORKSPACE_LIMIT_BYTES")
    assert ph["attn_hist"][0] == 1, ph
    assert binding.workspace_held_bytes() <= need
    o2, l2 = binding.forward(q, k, v, cu, B, topk)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_empty_batch():
    q = torch.empty((0, 4, 128), dtype=torch.bfloat16, device=DEV)
    k = torch.empty((0, 2, 128), dtype=torch.bfloat16, device=DEV)
    o, l = binding.forward(q, k, k, torch.tensor([0, 0], dtype=torch.int32), 64, 3)
    assert o.shape == (0, 4, 128) and l.shape == (4, 0)


def test_topk_covering_every_block_runs_the_dense_path():
    """top-k at least the longest sequence's block count selects every causal
    block (Eq. 5), so MoBA is full attention and the library runs the dense
    kernels: forward, backward and decode equal the dense calls bit for bit
    (the oracle comparisons of the cases with top-k > #blocks cover the
    values)."""
    q, k, v, cu = make((700, 300), 4, 2, torch.bfloat16, 128, offset=0.5, seed=37)  # 6 and 3 blocks
    o1, l1 = binding.forward(q, k, v, cu, 128, 6)
    o2, l2 = binding.dense_forward(q, k, v, cu)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    dout = inputs.make_dout(q.shape, q.dtype, 37, device=DEV)
    g1 = binding.backward(q, k, v, cu, 128, 6, o1, l1, dout)
    g2 = binding.dense_backward(q, k, v, cu, o2, l2, dout)
    for x, y in zip(g1, g2):
        assert torch.equal(x, y)
    qd = q[(cu[1:] - 1).to(torch.int64).to(DEV)].contiguous()
    d1 = binding.decode(qd, k, v, cu, 128, 6)
    d2 = binding.decode(qd, k, v, cu, 128, 0)
    assert torch.equal(d1[0], d2[0]) and torch.equal(d1[1], d2[1])
    # one block fewer than the longest sequence has: the MoBA kernels run
    o3, l3 = binding.forward(q, k, v, cu, 128, 5)
    assert not torch.equal(o3, o2)
