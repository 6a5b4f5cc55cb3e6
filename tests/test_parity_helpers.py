"""CPU checks of the comparison helpers in tests/parity.py that carry
arithmetic of their own.

delta_corrections: the backward forms each row's Delta = <dO, O> from the
rounded forward output it is given.  The exact gradients with that Delta are
computed here by brute force, key by key (softmax over the keys of Eq. 4,
dS = P (dP - Delta)), and must equal the oracle's gradients plus the
corrections.
"""
import math

import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2502_13189_amd import inputs
import parity


def brute_force_grads(Q, K, V, G, O, cu, B, sel):
    T, Hq, D = Q.shape
    Hkv = K.shape[1]
    s = 1.0 / np.sqrt(D)
    dq = np.zeros((T * Hq, D))
    dk = np.zeros_like(K)
    for t in range(T):
        sq = np.searchsorted(cu, t, side="right") - 1
        for h in range(Hq):
            r, g = t * Hq + h, h // (Hq // Hkv)
            keys = set()
            for b in sel[r]:
                if b >= 0:
                    keys.update(range(cu[sq] + b * B, min(cu[sq] + (b + 1) * B, t + 1)))
            keys = sorted(keys)
            z = np.array([Q[t, h] @ K[u, g] for u in keys]) * s
            p = np.exp(z - z.max())
            p /= p.sum()
            dp = np.array([G[t, h] @ V[u, g] for u in keys])
            ds = p * (dp - G[t, h] @ O[t, h])
            for j, u in enumerate(keys):
                dq[r] += s * ds[j] * K[u, g]
                dk[u, g] += s * ds[j] * Q[t, h]
    return dq, dk


@pytest.mark.parametrize("seqlens,hq,hkv,B,topk,seed", [
    ((40, 9), 2, 2, 1, 2, 210),      # one-key blocks: the deepest cancellation
    ((30, 0, 25), 4, 2, 8, 3, 5),    # an empty sequence, GQA groups of 2
])
def test_delta_corrections_match_brute_force(seqlens, hq, hkv, B, topk, seed):
    D = 32
    q, k, v, cu = inputs.make(seqlens, hq, hkv, D, torch.bfloat16, B, 0.5, seed)
    dout = inputs.make_dout(q.shape, q.dtype, seed)
    qn, kn, vn, dn = (inputs.to_oracle(x) for x in (q, k, v, dout))
    cun = cu.numpy()
    kbar = oracle.pool(kn, cun, B)
    sel = oracle.select(qn, kbar, cun, B, topk)
    odq, odk, _ = oracle.attend_backward(qn, kn, vn, dn, cun, B, sel, kv_window="all")
    oo, _ = oracle.attend(qn, kn, vn, cun, B, sel)
    T = q.shape[0]
    out = torch.tensor(oo.reshape(T, hq, D)).to(torch.bfloat16)
    ddq, ddk = parity.delta_corrections(q, k, v, cun, B, sel, out, dout, oo)
    bq, bk = brute_force_grads(*(x.double().numpy() for x in (q, k, v, dout, out)), cun, B, sel)
    # the rounding of O moves dq visibly; the correction takes it out exactly
    assert np.abs(bq - odq).max() > 1e3 * np.abs(bq - (odq + ddq)).max()
    assert np.abs(bq - (odq + ddq)).max() <= 1e-12 * np.abs(bq).max()
    # ddk goes through an fp32 upstream gradient: its rounding, 2^-24 relative
    assert np.abs(bk - (odk + ddk)).max() <= 1e-6 * np.abs(bk).max()


# ----------------------------------------------------------------------------
# the tie rule of the selection comparisons (Eq. 5 near ties)
# ----------------------------------------------------------------------------
TIE_B, TIE_K = 8, 3


def tie_case(seed=61, D=16):
    """Two sequences, 4 query / 2 kv heads, bf16.  In sequence 0 every block
    holds the same keys, so every gate score of a row ties exactly; sequence 1
    is Gaussian with per-block key offsets, where near ties are rare.  Values
    are 10 * (block index) plus noise, so attention over another block set
    moves the output far beyond the output tolerances."""
    q, k, v, cu = inputs.make((61, 70), 4, 2, D, torch.bfloat16, TIE_B, 0.5, seed)
    kk = k.clone()
    for t in range(61):
        kk[t] = k[t % TIE_B]
    vv = v.clone()
    for s, (a, b) in enumerate(((0, 61), (61, 131))):
        for t in range(a, b):
            vv[t] = v[t] * 0.1 + 10.0 * ((t - a) // TIE_B)
    return q, kk, vv.to(torch.bfloat16), cu


def np_scores(qn, kn, cu, B):
    """Block means, mean |K|, and every row's past-block scores (numpy fp64,
    independent of the oracle): {row: (scores [c], |q| . mean|K| [c])}."""
    qf, kf = parity._widen(qn), parity._widen(kn)
    T, Hq, D = qf.shape
    G = Hq // kf.shape[1]
    res = {}
    for s in range(len(cu) - 1):
        a, b = int(cu[s]), int(cu[s + 1])
        n = (b - a + B - 1) // B
        means = [kf[a + j * B:min(a + (j + 1) * B, b)].mean(0) for j in range(n)]
        absm = [np.abs(kf[a + j * B:min(a + (j + 1) * B, b)]).mean(0) for j in range(n)]
        for t in range(a, b):
            c = (t - a) // B
            for h in range(Hq):
                g = h // G
                res[t * Hq + h] = (np.array([qf[t, h] @ means[j][g] for j in range(c)]),
                                   np.array([np.abs(qf[t, h]) @ absm[j][g] for j in range(c)]))
    return res


def planted_swap(osel, i, out_block, in_block):
    row = [int(x) for x in osel[i] if x >= 0]
    c = row[-1]
    hist = sorted((set(row[:-1]) - {out_block}) | {in_block})
    new = np.full(osel.shape[1], -1, np.int32)
    new[:len(hist)] = hist
    new[len(hist)] = c
    return new


def test_check_selection_accepts_exact_ties_and_rejects_real_swaps():
    q, k, v, cu = tie_case()
    qn, kn = inputs.to_oracle(q), inputs.to_oracle(k)
    cun = cu.numpy()
    T, Hq, D = q.shape
    rows = np.arange(T * Hq, dtype=np.int64)
    osel = oracle.select(qn, oracle.pool(kn, cun, TIE_B), cun, TIE_B, TIE_K)
    sc = np_scores(qn, kn, cun, TIE_B)
    # exact ties (sequence 0, c >= k): the higher-index block in place of a
    # kept one is a correct selection and must be accepted
    g = osel.copy()
    tie_rows = [i for i in range(61 * Hq) if (i // Hq) // TIE_B >= TIE_K]
    for i in tie_rows:
        c = (i // Hq) // TIE_B
        g[i] = planted_swap(osel, i, int(osel[i][0]), c - 1)
    _, bad = parity.check_selection(g, rows, qn, kn, cun, TIE_B, TIE_K, exact=False)
    assert sorted(bad.tolist()) == tie_rows
    with pytest.raises(AssertionError):
        parity.check_selection(g, rows, qn, kn, cun, TIE_B, TIE_K, exact=True)
    _, bad = parity.check_selection_rows(g[rows], rows, qn.reshape(-1, D), T, Hq, kn, cun, TIE_B,
                                         TIE_K, exact=False)
    assert sorted(bad.tolist()) == tie_rows
    # a swap across a gap far above tau must be rejected, by both helpers
    n_checked = 0
    for r in range(61 * Hq, T * Hq):
        s, mag = sc[r]
        c = len(s)
        if c <= TIE_K:
            continue
        order = sorted(range(c), key=lambda j: (-s[j], j))
        a, b = order[TIE_K - 2], order[-1]   # the weakest kept and the worst dropped block
        tau = parity.TAU_SCALE * (mag[a] + mag[b])
        if s[a] - s[b] <= 100 * tau:
            continue
        g = osel.copy()
        g[r] = planted_swap(osel, r, a, b)
        with pytest.raises(AssertionError, match="score gap"):
            parity.check_selection(g[[r]], np.array([r]), qn, kn, cun, TIE_B, TIE_K, exact=False)
        with pytest.raises(AssertionError, match="score gap"):
            parity.check_selection_rows(g[[r]], np.array([r]), qn.reshape(-1, D)[[r]], T, Hq, kn,
                                        cun, TIE_B, TIE_K, exact=False)
        n_checked += 1
        if n_checked == 8:
            break
    assert n_checked == 8
    # a selection without its current block, or of the wrong size, is never a tie
    r = T * Hq - 1
    g = osel.copy()
    g[r][np.argmax(g[r])] -= 1
    with pytest.raises(AssertionError):
        parity.check_selection(g[[r]], np.array([r]), qn, kn, cun, TIE_B, TIE_K, exact=False)


def test_decode_ambiguous_rows_flags_exactly_the_near_ties():
    """decode_ambiguous_rows marks a row iff its (k-1)-th and k-th best past
    blocks (Eq. 5 order: score desc, index asc) are within tau of each other;
    recomputed here from numpy block means."""
    q, k, v, cu = tie_case(seed=67)
    qn, kn = inputs.to_oracle(q), inputs.to_oracle(k)
    cun = cu.numpy()
    T, Hq, D = q.shape
    rows = np.arange(T * Hq, dtype=np.int64)
    _, amb = parity.decode_ambiguous_rows(qn.reshape(-1, D), rows, T, Hq, kn, cun, TIE_B, TIE_K)
    sc = np_scores(qn, kn, cun, TIE_B)
    expect = np.zeros(len(rows), bool)
    for r in rows:
        s, mag = sc[int(r)]
        nh = min(TIE_K - 1, len(s))
        if nh == 0 or nh >= len(s):
            continue
        order = sorted(range(len(s)), key=lambda j: (-s[j], j))
        a, b = order[nh - 1], order[nh]
        expect[r] = s[a] - s[b] <= parity.TAU_SCALE * (mag[a] + mag[b])
    assert np.array_equal(amb, expect)
    assert expect[:61 * Hq].sum() > 100 and (~expect).sum() > 100


def test_admissible_selections_and_row_check():
    """Every exactly tied row of sequence 0 admits every choice of its k-1
    past blocks; Gaussian rows admit the oracle's alone.  Outputs over an
    admissible selection pass check_rows_any_selection; outputs over a block
    set beyond the tie bound fail it."""
    q, k, v, cu = tie_case(seed=71)
    qn, kn, vn = inputs.to_oracle(q), inputs.to_oracle(k), inputs.to_oracle(v)
    cun = cu.numpy()
    T, Hq, D = q.shape
    rows = np.arange(T * Hq, dtype=np.int64)
    qr = qn.reshape(-1, D)
    alts = parity.admissible_selections(qr, rows, T, Hq, kn, cun, TIE_B, TIE_K)
    for r in range(61 * Hq):
        c = (r // Hq) // TIE_B
        nh = min(TIE_K - 1, c)
        assert len(alts[r]) == math.comb(c, nh), (r, len(alts[r]))
        assert len({tuple(x) for x in alts[r]}) == len(alts[r])
    sc = np_scores(qn, kn, cun, TIE_B)
    n_single = sum(len(alts[r]) == 1 for r in range(61 * Hq, T * Hq))
    assert n_single > 0.9 * (T * Hq - 61 * Hq)
    # outputs over the last admissible selection of every row
    pick = np.stack([a[-1] for a in alts])
    oo, ol = oracle.attend(qn, kn, vn, cun, TIE_B, pick)
    mx, mean, lmx, multi, other = parity.check_rows_any_selection(oo, ol, qr, rows, T, Hq, kn, vn,
                                                                  cun, TIE_B, TIE_K)
    assert mx < 1e-12 and other > 100 and multi >= other
    # one Gaussian row computed over a block set beyond the tie bound
    for r in range(T * Hq - 1, 61 * Hq, -1):
        s, mag = sc[r]
        if len(s) > TIE_K and len(alts[r]) == 1:
            order = sorted(range(len(s)), key=lambda j: (-s[j], j))
            bad = planted_swap(alts[r][0][None], 0, order[TIE_K - 2], order[-1])
            break
    o1, l1 = oracle.attend_rows(qr[[r]], T, Hq, kn, vn, cun, TIE_B, bad[None], np.array([r]))
    with pytest.raises(AssertionError):
        parity.check_rows_any_selection(o1, l1, qr[[r]], np.array([r]), T, Hq, kn, vn, cun, TIE_B,
                                        TIE_K)


def test_tie_bound_is_applied_at_tau():
    """Gaps placed on either side of tau.  Three sequences of 257 tokens
    (B = 64, so the last token is in block 4, topk 3: two past blocks kept).
    Keys are 0 except dimension 0: 2 in block 0, 1 in block 2, 0 in block 3,
    and in block 1 the value 1 with m of its 64 tokens lowered to 1 - 2^-8
    (m = 1, 2, 3), so block 1 trails block 2 by m 2^-14.  The last query is
    e_0, so tau = 2^-14 (1 + 1 - m 2^-14): only m = 1 is within it."""
    B, K, D = 64, 3, 16
    L = 4 * B + 1
    T = 3 * L
    qf = np.zeros((T, 1, D), np.float32)
    kf = np.zeros((T, 1, D), np.float32)
    for s, m in enumerate((1, 2, 3)):
        a = s * L
        qf[a + L - 1, 0, 0] = 1.0
        kf[a:a + B, 0, 0] = 2.0
        kf[a + B:a + 2 * B, 0, 0] = 1.0
        kf[a + B:a + B + m, 0, 0] = 1.0 - 2.0 ** -8
        kf[a + 2 * B:a + 3 * B, 0, 0] = 1.0
    qn = (torch.from_numpy(qf).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16))
    kn = (torch.from_numpy(kf).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16))
    assert np.array_equal(parity._widen(kn), kf.astype(np.float64))
    cu = np.array([0, L, 2 * L, 3 * L], np.int32)
    rows = np.array([L - 1, 2 * L - 1, 3 * L - 1], np.int64)
    osel, amb = parity.decode_ambiguous_rows(qn.reshape(-1, D)[rows], rows, T, 1, kn, cu, B, K)
    assert [list(x) for x in osel] == [[0, 2, 4]] * 3
    assert amb.tolist() == [True, False, False]
    alts = parity.admissible_selections(qn.reshape(-1, D)[rows], rows, T, 1, kn, cu, B, K)
    assert [len(a) for a in alts] == [2, 1, 1]
    assert list(alts[0][1]) == [0, 1, 4]
    swapped = np.array([[0, 1, 4]] * 3, np.int32)
    _, bad = parity.check_selection(swapped[:1], rows[:1], qn, kn, cu, B, K, exact=False)
    assert bad.tolist() == [0]
    for i in (1, 2):
        with pytest.raises(AssertionError, match="score gap"):
            parity.check_selection(swapped[i:i + 1], rows[i:i + 1], qn, kn, cu, B, K, exact=False)
