"""Parity along the sweeps (Fig. 2a: block size 4096, top-12, 8K to 1M
tokens; Fig. 2b: 64 blocks per sequence, top-3, 8K to 10M tokens; block
granularity: 32K tokens at 75% sparsity, (B, k) = (4096, 2) .. (256, 32);
32 query / 8 kv heads, bf16), in the launch configuration the sweep times
(one moba_forward call per point).

Per length: the selection invariants on every row (on the GPU, token chunk by
token chunk); the tie-aware selection and the outputs on a sample of rows
(for every query head the block-boundary positions and 16 seeded uniform
positions, plus the last 256 tokens of head 0).  The oracle reads only the
sampled rows' query vectors, so K and V are the only full host copies.
The 4M, 8M and 10M-token points take most of the GPU's memory (at 10M: q
and out 82 GB each, k and v 20 GB each, the workspace under its 64 GiB cap)
and about a minute each.
"""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2502_13189_amd import binding, inputs
import parity

pytestmark = pytest.mark.gpu
DEV = "cuda:0"

CASES = [("fig2a", L, 4096) for L in (8192, 32768, 131072, 524288)] + \
        [("fig2b", L, L // 64) for L in (8192, 131072, 1048576, 2097152)] + \
        [("gran", 32768, B) for B in (4096, 2048, 1024, 512, 256)]
LARGE = [("fig2b", L, L // 64) for L in (4194304, 8388608, 10485760)]


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.load()


def sweep_rows(w, n_uniform=16, tail=256, seed=4321):
    B, k, L, Hq = w.block_size, w.topk, w.seqlens[0], w.hq
    rng = np.random.default_rng(seed)
    taus = {0, 1, B - 1, B, (k - 1) * B - 1, (k - 1) * B, k * B - 1, k * B, L // 2, L - B, L - 1}
    taus = {t for t in taus if 0 <= t < L}
    rows = set()
    for h in range(Hq):
        for t in taus | set(int(x) for x in rng.integers(0, L, size=n_uniform)):
            rows.add(t * Hq + h)
    for t in range(max(0, L - tail), L):
        rows.add(t * Hq)
    return np.array(sorted(rows), dtype=np.int64)


def selection_invariants_chunked(sel, B, topk, chunk=1 << 18):
    """Single sequence: on every row the current block c = t // B is selected,
    the history part is ascending below c with min(topk - 1, c) entries, and
    the rest is -1 padding."""
    T, Hq, K = sel.shape
    idx = torch.arange(K, device=sel.device)[None, None, :]
    for t0 in range(0, T, chunk):
        s = sel[t0:t0 + chunk].to(torch.int64)
        n = s.shape[0]
        c = (torch.arange(t0, t0 + n, device=sel.device) // B)[:, None].expand(n, Hq)
        nh = torch.clamp(c, max=topk - 1)
        assert torch.equal(torch.gather(s, 2, nh[..., None])[..., 0], c)
        hist = idx < nh[..., None]
        assert bool(((s < c[..., None]) & (s >= 0) | ~hist).all())
        if K > 1:
            assert bool(((s[..., 1:] > s[..., :-1]) | ~hist[..., 1:]).all())
        assert bool(((s == -1) | ~(idx > nh[..., None])).all())


def run_sweep_point(kind, L, B):
    w = inputs.sweep_workload(kind, L, B)
    # earlier calls' cached device memory (the library's workspace, torch's
    # free blocks) would not leave room for the largest points
    binding.release_workspace()
    torch.cuda.empty_cache()
    print("[sweep] %s: generating" % w.name, flush=True)
    q, k, v, cu = inputs.make_workload(w, device=DEV)
    print("[sweep] %s: forward and selection on the GPU" % w.name, flush=True)
    T, Hq, D = q.shape
    out, lse = binding.forward(q, k, v, cu, w.block_size, w.topk)
    sel = binding.select(q, k, cu, w.block_size, w.topk)
    torch.cuda.synchronize()
    selection_invariants_chunked(sel, w.block_size, w.topk)
    rows = sweep_rows(w)
    rows_t = torch.as_tensor(rows, device=DEV)
    q_rows = inputs.to_oracle(q.view(T * Hq, D)[rows_t])
    gsel = sel.view(T * Hq, w.topk)[rows_t].cpu().numpy()
    gout, glse = parity.gather_rows(out, lse, rows)
    del q, out, sel
    kn, vn = inputs.to_oracle(k), inputs.to_oracle(v)
    del k, v, lse
    torch.cuda.empty_cache()
    cun = cu.numpy()
    print("[sweep] %s: oracle on %d rows" % (w.name, len(rows)), flush=True)
    osel, bad = parity.check_selection_rows(gsel, rows, q_rows, T, Hq, kn, cun, w.block_size,
                                            w.topk, exact=False)
    use = osel.copy()
    use[bad] = gsel[bad]
    oout, olse = oracle.attend_rows(q_rows, T, Hq, kn, vn, cun, w.block_size, use, rows)
    mx, mean, lmx = parity.compare_outputs(gout, glse, oout, olse, "bf16", w.name)
    print("%s: rows %d (tie-explained %d), out max-abs %.2e mean-abs %.2e, lse %.2e"
          % (w.name, len(rows), len(bad), mx, mean, lmx))


@pytest.mark.parametrize("kind,L,B", CASES, ids=["%s_L%d_B%d" % c for c in CASES])
def test_sweep_parity(kind, L, B):
    run_sweep_point(kind, L, B)


@pytest.mark.parametrize("kind,L,B", LARGE, ids=["%s_L%d_B%d" % c for c in LARGE])
def test_sweep_parity_large(kind, L, B):
    run_sweep_point(kind, L, B)
