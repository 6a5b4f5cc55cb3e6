"""Comparison helpers for the GPU parity tests: run the library and the fp64
oracle on the same inputs and compare selections and outputs.

Selection rule.  On fp32 inputs the selection must equal the oracle's
exactly.  On bf16 inputs the fp32 gate may order two blocks whose exact
scores are closer than its rounding error differently from the fp64 oracle;
such a row is accepted iff every block the GPU kept instead of an oracle block
is tie-explained: s_oracle_block - s_gpu_block <= tau_a + tau_b, with
tau_j = 2^-14 * sum_i |q_i| * mean_over_block(|K[., g, i]|) (a bound on the
fp32 rounding of the block mean and the 128-term dot product, with margin).
Outputs of tie-explained rows are compared with the oracle's attention over
the GPU's own selection.
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import oracle
from paper_2502_13189_amd import binding, inputs

TAU_SCALE = 2.0 ** -14

# output tolerances: max-abs and mean-abs for bf16; max-abs for fp32
BF16_MAX_ABS, BF16_MEAN_ABS = 2e-2, 2e-3
F32_MAX_ABS = 1e-4
LSE_ABS = {"bf16": 1e-3, "f32": 1e-5}


def host_inputs(q, k, v):
    return inputs.to_oracle(q), inputs.to_oracle(k), inputs.to_oracle(v)


def block_offsets(cu, B):
    cu = list(cu)
    off, acc = [], 0
    for s in range(len(cu) - 1):
        off.append(acc)
        acc += (cu[s + 1] - cu[s] + B - 1) // B
    return off


def seq_of_tokens(cu, t):
    cu = np.asarray(cu)
    return np.searchsorted(cu, t, side="right") - 1


def check_selection(gpu_sel, rows, qn, kn, cu, B, topk, exact, pooled=None):
    """Compare GPU selections (for `rows`) with the oracle's.  Returns
    (oracle_sel, mismatch_rows).  Raises AssertionError on a mismatch that is
    not allowed.  pooled: the oracle's (block means, mean |K|) of kn, if
    already computed."""
    cu = np.asarray(cu)
    kbar, kabs = pooled if pooled is not None else oracle.pool(kn, cu, B, with_abs=True)
    osel = oracle.select(qn, kbar, cu, B, topk, rows=rows)
    gsel = np.asarray(gpu_sel).reshape(len(rows), topk)
    bad = np.nonzero((gsel != osel).any(axis=1))[0]
    if exact:
        assert bad.size == 0, "selection differs on %d rows, first rows %s" % (bad.size, rows[bad[:5]])
        return osel, bad
    if bad.size == 0:
        return osel, bad
    Hq = qn.shape[1]
    G = Hq // kn.shape[1]
    nmax = int(max(osel.max(), gsel.max())) + 1
    _, sc = oracle.select(qn, kbar, cu, B, topk, rows=rows[bad], nmax=nmax)
    boff = block_offsets(cu, B)
    qf = np.abs(_widen(qn))
    af = kabs
    for n, i in enumerate(bad):
        r = int(rows[i])
        t, h = r // Hq, r % Hq
        g = h // G
        s = int(seq_of_tokens(cu, t))
        o_set = set(int(x) for x in osel[i] if x >= 0)
        g_set = set(int(x) for x in gsel[i] if x >= 0)
        assert len(o_set) == len(g_set) and max(o_set) == max(g_set), (r, o_set, g_set)
        for jg in g_set - o_set:
            for jo in o_set - g_set:
                tau = TAU_SCALE * (qf[t, h] @ af[boff[s] + jg, g] + qf[t, h] @ af[boff[s] + jo, g])
                gap = sc[n, jo] - sc[n, jg]
                assert gap <= tau, ("row %d: GPU kept block %d over block %d, score gap %.3e > "
                                    "tolerance %.3e" % (r, jg, jo, gap, tau))
    return osel, bad


def check_selection_rows(gpu_sel, rows, q_rows, T, Hq, kn, cu, B, topk, exact):
    """check_selection() for problems too large to copy whole: q_rows holds
    only the listed rows' query vectors [nrows, D] (list order)."""
    cu = np.asarray(cu)
    kbar, kabs = oracle.pool(kn, cu, B, with_abs=True)
    osel = oracle.select_rows(q_rows, T, Hq, kbar, cu, B, topk, rows)
    gsel = np.asarray(gpu_sel).reshape(len(rows), topk)
    bad = np.nonzero((gsel != osel).any(axis=1))[0]
    if exact:
        assert bad.size == 0, "selection differs on %d rows, first rows %s" % (bad.size, rows[bad[:5]])
        return osel, bad
    if bad.size == 0:
        return osel, bad
    G = Hq // kn.shape[1]
    nmax = int(max(osel.max(), gsel.max())) + 1
    _, sc = oracle.select_rows(q_rows[bad], T, Hq, kbar, cu, B, topk, rows[bad], nmax=nmax)
    boff = block_offsets(cu, B)
    qf = np.abs(_widen(np.asarray(q_rows).reshape(len(rows), -1)))
    for n, i in enumerate(bad):
        r = int(rows[i])
        t, h = r // Hq, r % Hq
        g = h // G
        s = int(seq_of_tokens(cu, t))
        o_set = set(int(x) for x in osel[i] if x >= 0)
        g_set = set(int(x) for x in gsel[i] if x >= 0)
        assert len(o_set) == len(g_set) and max(o_set) == max(g_set), (r, o_set, g_set)
        for jg in g_set - o_set:
            for jo in o_set - g_set:
                tau = TAU_SCALE * (qf[i] @ kabs[boff[s] + jg, g] + qf[i] @ kabs[boff[s] + jo, g])
                gap = sc[n, jo] - sc[n, jg]
                assert gap <= tau, ("row %d: GPU kept block %d over block %d, score gap %.3e > "
                                    "tolerance %.3e" % (r, jg, jo, gap, tau))
    return osel, bad


def _widen(x):
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


def compare_outputs(gout, glse, oout, olse, dtype, what=""):
    gout = np.asarray(gout, dtype=np.float64)
    err = np.abs(gout - oout)
    lerr = np.abs(np.asarray(glse, np.float64) - olse)
    if dtype == "f32":
        assert err.max() <= F32_MAX_ABS, "%s out max-abs %.3e" % (what, err.max())
    else:
        assert err.max() <= BF16_MAX_ABS, "%s out max-abs %.3e" % (what, err.max())
        assert err.mean() <= BF16_MEAN_ABS, "%s out mean-abs %.3e" % (what, err.mean())
    assert lerr.max() <= LSE_ABS[dtype], "%s lse max-abs %.3e" % (what, lerr.max())
    return float(err.max()), float(err.mean()), float(lerr.max())


def gather_rows(out, lse, rows):
    """Rows (t*Hq+h) of a GPU output [T, Hq, D] and lse [Hq, T], on the host."""
    T, Hq, D = out.shape
    rows_t = torch.as_tensor(rows, dtype=torch.int64, device=out.device)
    t, h = rows_t // Hq, rows_t % Hq
    o = out[t, h].float().cpu().numpy()
    l = lse[h, t].float().cpu().numpy()
    return o, l


def moba_parity(q, k, v, cu, B, topk, rows=None, dtype="bf16", exact_sel=None):
    """Run the library and the oracle; assert selection and output parity on
    `rows` (all rows if None).  Returns a dict of error figures."""
    cu_t = cu if isinstance(cu, torch.Tensor) else torch.tensor(cu, dtype=torch.int32)
    out, lse = binding.forward(q, k, v, cu_t, B, topk)
    gsel_full = binding.select(q, k, cu_t, B, topk)
    torch.cuda.synchronize()
    T, Hq, D = q.shape
    if rows is None:
        rows = np.arange(T * Hq, dtype=np.int64)
    qn, kn, vn = host_inputs(q, k, v)
    cun = cu_t.numpy()
    rows_t = torch.as_tensor(rows, device=q.device)
    gsel = gsel_full.view(T * Hq, topk)[rows_t].cpu().numpy()
    exact = (dtype == "f32") if exact_sel is None else exact_sel
    osel, bad = check_selection(gsel, rows, qn, kn, cun, B, topk, exact)
    use_sel = osel.copy()
    use_sel[bad] = gsel[bad]
    oout, olse = oracle.attend(qn, kn, vn, cun, B, use_sel, rows=rows)
    gout, glse = gather_rows(out, lse, rows)
    mx, mean, lmx = compare_outputs(gout, glse, oout, olse, dtype)
    return {"rows": len(rows), "tie_rows": int(bad.size), "max_abs": mx, "mean_abs": mean,
            "lse_max_abs": lmx, "out": out, "lse": lse, "sel": gsel_full}


def dense_parity(q, k, v, cu, rows=None, dtype="bf16"):
    cu_t = cu if isinstance(cu, torch.Tensor) else torch.tensor(cu, dtype=torch.int32)
    out, lse = binding.dense_forward(q, k, v, cu_t)
    torch.cuda.synchronize()
    T, Hq, D = q.shape
    if rows is None:
        rows = np.arange(T * Hq, dtype=np.int64)
    qn, kn, vn = host_inputs(q, k, v)
    oout, olse = oracle.dense(qn, kn, vn, cu_t.numpy(), rows=rows)
    gout, glse = gather_rows(out, lse, rows)
    mx, mean, lmx = compare_outputs(gout, glse, oout, olse, dtype, "dense")
    return {"rows": len(rows), "max_abs": mx, "mean_abs": mean, "lse_max_abs": lmx}


# Backward tolerances (bf16).  bf16 rounding has unit roundoff u = 2^-8.  The
# kernels round each P and dS term to bf16 once (<= u relative), use Delta =
# <dO, O> with the forward's bf16 O (whose error stays within ~3u per element
# after the partial rounding and the merge), accumulate in fp32 (negligible
# here) and round the result once (<= u).  So every gradient element obeys
#   |err| <= 3u (|ref| + c),
# c the oracle's sum of absolute terms (cq, ck, cv of attend_backward); the
# elementwise bound below is 4u.  It is a worst case; a systematic error (a
# dropped block, a wrong mask) shows in the mean instead, bounded by
# BWD_MEAN_REL = 2u of the mean |ref| (the mean error observed is about
# 0.65u, mostly the final rounding).
#
# The mean check compares with the exact gradients evaluated with the Delta
# that the rounded O gives (delta_corrections below), not with the oracle's
# exact Delta.  On rows with few keys dq and dk cancel deeply (c >> |ref|),
# and the rounding of O, an input of the backward, alone moves their mean by
# more than 2u of the small mean |ref|; dq and dk are linear in Delta, so the
# evaluation with the rounded O's Delta is exact, and what remains is the
# kernels' own arithmetic.
BWD_ELEM_U = 4.0 * 2.0 ** -8
BWD_MEAN_REL = 2.0 ** -7


def delta_corrections(q, k, v, cu, B, sel, out, dout, o_exact):
    """Changes of the exact dq and dk when each row's Delta = <dO, O> is
    taken from the rounded forward output `out` instead of the exact O.
    With dS = P (dP - Delta), dq_i = s sum_u dS_iu k_u and dk_u = s sum_i dS_iu
    q_i (s = 1/sqrt(D)), a change d_i of Delta_i moves dq_i by -s d_i sum_u P_iu
    k_u (attention with the keys as values) and dk_u by -s sum_i P_iu d_i q_i
    (the dV of an upstream gradient d_i q_i).  Both come from the oracle.
    Returns (ddq [rows, D], ddk [T, Hkv, D])."""
    T, Hq, D = q.shape
    s = 1.0 / np.sqrt(D)
    og = out.float().cpu().numpy().astype(np.float64).reshape(o_exact.shape)
    gd = dout.float().cpu().numpy().astype(np.float64).reshape(o_exact.shape)
    d = (gd * (og - o_exact)).sum(-1)
    qf, kf, vf = (x.float().cpu().numpy() for x in (q, k, v))
    a, _ = oracle.attend(qf, kf, kf, cu, B, sel)
    ddq = -s * d[:, None] * a
    up = (d[:, None] * qf.reshape(-1, D).astype(np.float64)).astype(np.float32).reshape(q.shape)
    _, _, pv = oracle.attend_backward(qf, kf, vf, up, cu, B, sel, want_dq=False, kv_window="all")
    return ddq, -s * pv


def moba_backward_parity(q, k, v, cu, B, topk, dout, exact_sel=False):
    """Run forward + backward on the GPU and the oracle's fp64 gradients on the
    selection the GPU made (oracle selection; tie-explained rows take the GPU's
    order, as in moba_parity).  Asserts the backward tolerances and returns,
    per gradient, (max of |err| / (|ref| + c), mean |err| / mean |ref|)."""
    cu_t = cu if isinstance(cu, torch.Tensor) else torch.tensor(cu, dtype=torch.int32)
    out, lse = binding.forward(q, k, v, cu_t, B, topk)
    dq, dk, dv = binding.backward(q, k, v, cu_t, B, topk, out, lse, dout)
    gsel = binding.select(q, k, cu_t, B, topk)
    torch.cuda.synchronize()
    T, Hq, D = q.shape
    Hkv = k.shape[1]
    rows = np.arange(T * Hq, dtype=np.int64)
    qn, kn, vn = host_inputs(q, k, v)
    dn = inputs.to_oracle(dout)
    cun = cu_t.numpy()
    gs = gsel.view(T * Hq, topk).cpu().numpy()
    osel, bad = check_selection(gs, rows, qn, kn, cun, B, topk, exact_sel)
    use_sel = osel.copy()
    use_sel[bad] = gs[bad]
    odq, odk, odv, cq, ck, cv = oracle.attend_backward(qn, kn, vn, dn, cun, B, use_sel,
                                                       kv_window="all", with_bounds=True)
    oo, _ = oracle.attend(qn, kn, vn, cun, B, use_sel)
    ddq, ddk = delta_corrections(q, k, v, cun, B, use_sel, out, dout, oo)
    res = {"tie_rows": int(bad.size)}
    for name, g, ref, c, dd in (("dq", dq, odq, cq, ddq), ("dk", dk, odk, ck, ddk),
                                ("dv", dv, odv, cv, 0.0)):
        g = g.float().cpu().numpy().astype(np.float64).reshape(ref.shape)
        assert np.isfinite(g).all(), "%s has non-finite values" % name
        err = np.abs(g - ref)
        ratio = err / (np.abs(ref) + c + 1e-30)
        worst = np.unravel_index(int(np.argmax(ratio)), ratio.shape)
        mean_rel = float(np.abs(g - (ref + dd)).mean() / max(np.abs(ref).mean(), 1e-30))
        res[name] = (float(ratio.max()), mean_rel)
        assert ratio.max() <= BWD_ELEM_U, ("%s element %s: |err| %.3e > %.3g (|ref| + c) with ref "
                                           "%.3e, c %.3e" % (name, worst, err[worst], BWD_ELEM_U,
                                                             ref[worst], c[worst]))
        assert mean_rel <= BWD_MEAN_REL, "%s mean |err| %.3e of mean |ref|" % (name, mean_rel)
    return res


def decode_ambiguous_rows(q_rows, rows, T, Hq, kn, cu, B, topk):
    """Decode rows (given by their query vectors q_rows and row ids) whose
    oracle top-(k-1) boundary is within the gate's rounding bound, where two
    selections are correct.  Returns (oracle selection, ambiguous mask)."""
    kbar, kabs = oracle.pool(kn, cu, B, with_abs=True)
    osel = oracle.select_rows(q_rows, T, Hq, kbar, cu, B, topk, rows)
    nmax = int(osel.max()) + 2
    _, sc = oracle.select_rows(q_rows, T, Hq, kbar, cu, B, topk, rows, nmax=nmax)
    qf = np.abs(_widen(np.asarray(q_rows).reshape(len(rows), -1)))
    boff = block_offsets(cu, B)
    G = Hq // kn.shape[1]
    amb = np.zeros(len(rows), bool)
    for i, r in enumerate(rows):
        t, h = int(r) // Hq, int(r) % Hq
        s = int(seq_of_tokens(cu, t))
        c = (t - int(cu[s])) // B
        nh = min(topk - 1, c)
        if nh == 0 or nh >= c:
            continue
        cand = sc[i, :c]
        order = sorted(range(c), key=lambda j: (-cand[j], j))
        ja, jb = order[nh - 1], order[nh]
        tau = TAU_SCALE * (qf[i] @ kabs[boff[s] + ja, h // G] + qf[i] @ kabs[boff[s] + jb, h // G])
        amb[i] = cand[ja] - cand[jb] <= tau
    return osel, amb


def admissible_selections(q_rows, rows, T, Hq, kn, cu, B, topk, max_swap=3):
    """Every selection a correct fp32 gate may return for each listed row
    (query vectors q_rows [nrows, D] in list order).  Eq. 5 orders the past
    blocks by exact score; the gate's rounding may reorder two blocks a, b
    whose exact scores differ by at most tau_a + tau_b (the bound of
    check_selection).  So a selection is admissible iff every block it keeps
    and every past block it drops are in Eq. 5's order up to that bound.
    Returns one list per row, the oracle's selection first, then the
    admissible ones reached by exchanging up to max_swap kept blocks with
    dropped ones near the boundary."""
    import itertools

    cu = np.asarray(cu)
    kbar, kabs = oracle.pool(kn, cu, B, with_abs=True)
    osel = oracle.select_rows(q_rows, T, Hq, kbar, cu, B, topk, rows)
    boff = block_offsets(cu, B)
    G = Hq // kn.shape[1]
    cs = []
    for r in rows:
        t = int(r) // Hq
        s = int(seq_of_tokens(cu, t))
        cs.append((t - int(cu[s])) // B)
    nmax = max(cs) + 1 if len(cs) else 1
    _, sc = oracle.select_rows(q_rows, T, Hq, kbar, cu, B, topk, rows, nmax=nmax)
    qf = np.abs(_widen(np.asarray(q_rows).reshape(len(rows), -1)))
    result = []
    for i, r in enumerate(rows):
        t, h = int(r) // Hq, int(r) % Hq
        s = int(seq_of_tokens(cu, t))
        c = cs[i]
        alts = [osel[i].copy()]
        nh = min(topk - 1, c)
        if 0 < nh < c:
            tau = TAU_SCALE * (kabs[boff[s]:boff[s] + c, h // G] @ qf[i])
            score = sc[i, :c]
            kept = [int(x) for x in osel[i][:nh]]
            dropped = [j for j in range(c) if j not in set(kept)]

            def near(a, b):
                return score[b] - score[a] <= tau[a] + tau[b] and score[a] - score[b] <= tau[a] + tau[b]

            kin = [a for a in kept if any(near(a, b) for b in dropped)]
            kout = [b for b in dropped if any(near(a, b) for a in kept)]
            for n in range(1, min(max_swap, len(kin), len(kout)) + 1):
                for xs in itertools.combinations(kin, n):
                    for ys in itertools.combinations(kout, n):
                        keep = sorted((set(kept) - set(xs)) | set(ys))
                        drop = [j for j in range(c) if j not in set(keep)]
                        if all(score[b] - score[a] <= tau[a] + tau[b] for a in keep for b in drop):
                            alt = np.full(topk, -1, np.int32)
                            alt[:nh] = keep
                            alt[nh] = c
                            alts.append(alt)
        result.append(alts)
    return result


def check_rows_any_selection(gout, glse, q_rows, rows, T, Hq, kn, vn, cu, B, topk, what=""):
    """Outputs of rows whose selection is not returned (decode): each row must
    match the oracle's attention over one of its admissible selections
    (admissible_selections); the row's closest one is used for the
    tolerances of compare_outputs.  Returns (max-abs, mean-abs, lse max-abs,
    rows with several admissible selections, rows matched by one other than
    the oracle's)."""
    alts = admissible_selections(q_rows, rows, T, Hq, kn, cu, B, topk)
    idx = np.array([i for i, a in enumerate(alts) for _ in a], np.int64)
    sels = np.stack([x for a in alts for x in a]) if len(idx) else np.zeros((0, topk), np.int32)
    qr = np.asarray(q_rows).reshape(len(rows), -1)
    oo, ol = oracle.attend_rows(qr[idx], T, Hq, kn, vn, np.asarray(cu), B, sels, np.asarray(rows)[idx])
    gout = np.asarray(gout, np.float64).reshape(len(rows), -1)
    glse = np.asarray(glse, np.float64).reshape(len(rows))
    best_o = np.empty_like(gout)
    best_l = np.empty_like(glse)
    pos, multi, other = 0, 0, 0
    for i, a in enumerate(alts):
        n = len(a)
        err = [np.abs(gout[i] - oo[pos + x]).max() + np.abs(glse[i] - ol[pos + x]) for x in range(n)]
        x = int(np.argmin(err))
        best_o[i], best_l[i] = oo[pos + x], ol[pos + x]
        multi += n > 1
        other += x > 0
        pos += n
    mx, mean, lmx = compare_outputs(gout, glse, best_o, best_l, "bf16", what)
    return mx, mean, lmx, multi, other
