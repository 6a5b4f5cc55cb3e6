"""CPU checks of the comparison helpers in tests/parity.py that carry
arithmetic of their own.

delta_corrections: the backward forms each row's Delta = <dO, O> from the
rounded forward output it is given.  The exact gradients with that Delta are
computed here by brute force, key by key (softmax over the keys of Eq. 4,
dS = P (dP - Delta)), and must equal the oracle's gradients plus the
corrections.
"""
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
