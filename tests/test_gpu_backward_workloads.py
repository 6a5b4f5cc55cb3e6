"""Backward parity at full workload sizes, in the launch configuration that
`bench.py --backward` times (one moba_forward for out/lse, one moba_backward).

Too large for the oracle to produce every gradient, so per workload:
  - dQ on a sample of rows (every query head at the sequence starts, block
    boundaries and ends, plus seeded uniform tokens), against the oracle's
    gradients for those rows alone (its attention reads only their vectors);
  - dK and dV exactly on the last 64 keys of every sequence and kv-head: they
    sit in the sequence's last block, which is never a history block, so only
    the block's own rows at or after each key attend them;
  - on every key, the identities that hold at any size: per sequence and
    kv-head the dK sum to zero and the dV sum to the summed upstream
    gradients of the group's query heads (softmax weights of a row sum to one).
The elementwise and mean tolerances are those of tests/parity.py; the sum
identities are checked against the size of the rounding noise of the summed
bf16 gradients (see check_sums).
"""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2502_13189_amd import binding, inputs
import parity

pytestmark = pytest.mark.gpu
DEV = "cuda:0"

WORKLOADS = ["bf16_L32k_gqa32x8_B2048_k3", "bf16_varlen4_T111920_mha32_B1024_k4",
             "bf16_L1M_gqa32x8_B4096_k12"]
TAIL = 64


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    binding.load()


def sample_rows(w, cu, n_uniform=24, seed=2468):
    B, Hq = w.block_size, w.hq
    T = int(cu[-1])
    rng = np.random.default_rng(seed)
    toks = set(int(x) for x in rng.integers(0, T, size=n_uniform))
    for s in range(len(cu) - 1):
        a, b = int(cu[s]), int(cu[s + 1])
        for t in (a, a + 1, a + B - 1, a + B, a + (w.topk - 1) * B, a + w.topk * B, b - B, b - 1):
            if a <= t < b:
                toks.add(t)
    return np.array(sorted(t * Hq + h for t in toks for h in range(Hq)), dtype=np.int64)


def compare(name, g, ref, c):
    g = np.asarray(g, np.float64).reshape(ref.shape)
    err = np.abs(g - ref)
    ratio = err / (np.abs(ref) + c + 1e-30)
    mean_rel = float(err.mean() / max(np.abs(ref).mean(), 1e-30))
    assert np.isfinite(g).all(), name
    assert ratio.max() <= parity.BWD_ELEM_U, "%s: |err| %.3g (|ref| + c) at %s" % (
        name, ratio.max(), np.unravel_index(int(np.argmax(ratio)), ratio.shape))
    assert mean_rel <= parity.BWD_MEAN_REL, "%s: mean |err| %.3e of mean |ref|" % (name, mean_rel)
    return float(ratio.max()), mean_rel


def check_sums(dk, dv, dout, cu, G, chunk=1 << 16):
    """Per sequence and kv-head: sum_t dk = 0 and sum_t dv = sum over the
    group's heads of sum_t dout.  Exact in real arithmetic; each bf16 gradient
    element carries its own rounding noise of a few u of the terms it sums, so
    the residual of a sum over n elements is compared with 16 u times the root
    of the sum of squares of what is summed (a dropped row or key
    contribution leaves a residual of the size of the terms themselves).
    Returns the largest residual / bound ratio (<= 1 passes)."""
    u = 2.0 ** -8
    worst = 0.0
    for s in range(len(cu) - 1):
        a, b = int(cu[s]), int(cu[s + 1])
        if b == a:
            continue
        Hkv, D = dk.shape[1], dk.shape[2]
        sk = torch.zeros(Hkv, D, dtype=torch.float64, device=dk.device)
        qk = torch.zeros_like(sk)
        sv = torch.zeros_like(sk)
        qv = torch.zeros_like(sk)
        so = torch.zeros_like(sk)
        for t0 in range(a, b, chunk):
            t1 = min(b, t0 + chunk)
            k64, v64 = dk[t0:t1].double(), dv[t0:t1].double()
            o64 = dout[t0:t1].double().view(t1 - t0, Hkv, G, D)
            sk += k64.sum(0)
            qk += (k64 * k64).sum(0)
            sv += v64.sum(0)
            qv += (v64 * v64).sum(0)
            so += o64.sum(dim=(0, 2))
        rk = sk.abs() / (16 * u * qk.sqrt() + 1e-30)
        rv = (sv - so).abs() / (16 * u * qv.sqrt() + 1e-30)
        worst = max(worst, float(rk.max()), float(rv.max()))
    return worst


@pytest.mark.parametrize("name", WORKLOADS)
def test_backward_workload(name):
    w = inputs.WORKLOADS[name]
    print("[bwd] %s: generating" % name, flush=True)
    q, k, v, cu = inputs.make_workload(w, device=DEV)
    dout = inputs.make_dout(q.shape, q.dtype, w.seed, device=DEV)
    T, Hq, D = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    print("[bwd] %s: forward, backward, selection on the GPU" % name, flush=True)
    out, lse = binding.forward(q, k, v, cu, w.block_size, w.topk)
    dq, dk, dv = binding.backward(q, k, v, cu, w.block_size, w.topk, out, lse, dout)
    sel = binding.select(q, k, cu, w.block_size, w.topk)
    torch.cuda.synchronize()
    cun = cu.numpy()

    worst_sum = check_sums(dk, dv, dout, cun, G)
    print("[bwd] %s: sum identities at %.3f of their bound" % (name, worst_sum), flush=True)

    rows = sample_rows(w, cun)
    tails = []
    for s in range(len(cun) - 1):
        a, b = int(cun[s]), int(cun[s + 1])
        if b == a:
            continue
        last0 = a + (b - a - 1) // w.block_size * w.block_size
        tails.append((max(last0, b - TAIL), b))
    trows = np.array(sorted(t * Hq + h for (k0, k1) in tails for t in range(k0, k1) for h in range(Hq)),
                     dtype=np.int64)

    def host_rows(x, r):
        rt = torch.as_tensor(r, device=DEV)
        return inputs.to_oracle(x.reshape(T * Hq, D)[rt])

    q_r, d_r = host_rows(q, rows), host_rows(dout, rows)
    q_t, d_t = host_rows(q, trows), host_rows(dout, trows)
    rt = torch.as_tensor(rows, device=DEV)
    tt = torch.as_tensor(trows, device=DEV)
    gs_r = sel.view(T * Hq, w.topk)[rt].cpu().numpy()
    gs_t = sel.view(T * Hq, w.topk)[tt].cpu().numpy()
    gdq = dq.reshape(T * Hq, D)[rt].float().cpu().numpy()
    gdk = [dk[k0:k1].float().cpu().numpy() for (k0, k1) in tails]
    gdv = [dv[k0:k1].float().cpu().numpy() for (k0, k1) in tails]
    del q, out, lse, dout, dq, dk, dv, sel
    kn, vn = inputs.to_oracle(k), inputs.to_oracle(v)
    del k, v
    torch.cuda.empty_cache()

    print("[bwd] %s: oracle dQ on %d rows" % (name, len(rows)), flush=True)
    osel, bad = parity.check_selection_rows(gs_r, rows, q_r, T, Hq, kn, cun, w.block_size, w.topk,
                                            exact=False)
    use = osel.copy()
    use[bad] = gs_r[bad]
    odq, _, _, cq, _, _ = oracle.attend_backward(q_r, kn, vn, d_r, cun, w.block_size, use,
                                                 rows=rows, shape=(T, Hq), with_bounds=True)
    rq = compare("dq", gdq, odq, cq)

    print("[bwd] %s: oracle dK/dV on the last %d keys of each sequence (%d rows)" %
          (name, TAIL, len(trows)), flush=True)
    osel_t, bad_t = parity.check_selection_rows(gs_t, trows, q_t, T, Hq, kn, cun, w.block_size,
                                                w.topk, exact=False)
    use_t = osel_t.copy()
    use_t[bad_t] = gs_t[bad_t]
    rk = rv = (0.0, 0.0)
    for i, (k0, k1) in enumerate(tails):
        sel_rows = (trows // Hq >= k0) & (trows // Hq < k1)
        _, odk, odv, _, ck, cv = oracle.attend_backward(
            q_t[sel_rows], kn, vn, d_t[sel_rows], cun, w.block_size, use_t[sel_rows],
            rows=trows[sel_rows], shape=(T, Hq), want_dq=False, kv_window=(k0, k1), with_bounds=True)
        a = compare("dk", gdk[i], odk, ck)
        b = compare("dv", gdv[i], odv, cv)
        rk = (max(rk[0], a[0]), max(rk[1], a[1]))
        rv = (max(rv[0], b[0]), max(rv[1], b[1]))
    print("%s: dq rows %d (tie-explained %d) %.2e/%.2e; tail dk %.2e/%.2e dv %.2e/%.2e "
          "(max |err|/(|ref|+c), mean |err|/mean |ref|); sum identities at %.2f of their bound"
          % (name, len(rows), len(bad), rq[0], rq[1], rk[0], rk[1], rv[0], rv[1], worst_sum))
    assert worst_sum <= 1.0, "sum identities: residual %.3f of the rounding-noise bound" % worst_sum
