"""Seeded synthetic inputs for MoBA prefill workloads.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic.  Both the GPU library and the fp64 oracle are fed from it.

The paper measures prefill on real long-context text through Llama-3.1-8B
(Sec. 3.3-3.4); no such data or weights exist here, so every workload is seeded
Gaussian data with the paper's shapes (heads, head_dim, block size, top-k,
lengths):

  * Q, K, V entries i.i.d. N(0, 1), drawn in that order, fp32;
  * optionally a per-(sequence block, kv-head) offset vector with entries
    N(0, key_offset_std^2), drawn after V and added in fp32 to every key of
    that block (this gives the gate something to find);
  * bf16 workloads round the fp32 draws once, to nearest-even.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch


@dataclass(frozen=True)
class Workload:
    name: str
    seqlens: tuple
    hq: int
    hkv: int
    d: int
    dtype: str  # "f32" or "bf16"
    block_size: int
    topk: int
    key_offset_std: float = 0.0
    seed: int = 0
    note: str = field(default="", compare=False)

    @property
    def total_tokens(self) -> int:
        return int(sum(self.seqlens))

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16


# The five prefill workloads: the shapes of the paper's settings (8K/B=512/top-3
# scaling-law runs, 32K/B=2048/top-3 hybrid runs, 1M/B=4096/top-12 long-context
# model) plus a tiny fp32 case and a ragged packed batch.
WORKLOADS = {
    w.name: w
    for w in [
        Workload("f32_L1k_h1_B128_k3", (1024,), 1, 1, 128, "f32", 128, 3, 0.0, 1,
                 "single causal sequence, fp32, 8 blocks"),
        Workload("bf16_L8k_mha32_B512_k3", (8192,), 32, 32, 128, "bf16", 512, 3, 0.5, 2,
                 "8K prefill, MHA, per-block key offsets"),
        Workload("bf16_L32k_gqa32x8_B2048_k3", (32768,), 32, 8, 128, "bf16", 2048, 3, 0.0, 3,
                 "32K prefill, GQA 32/8"),
        Workload("bf16_varlen4_T111920_mha32_B1024_k4", (4096, 12288, 30000, 65536), 32, 32, 128,
                 "bf16", 1024, 4, 0.0, 4, "packed batch of 4 ragged sequences"),
        Workload("bf16_L1M_gqa32x8_B4096_k12", (1048576,), 32, 8, 128, "bf16", 4096, 12, 0.5, 5,
                 "1M-token prefill, GQA 32/8, per-block key offsets"),
    ]
}

# The 1M-token workload is the one the throughput figure is quoted on.
HEADLINE = "bf16_L1M_gqa32x8_B4096_k12"


def cu_seqlens(seqlens) -> torch.Tensor:
    """Prefix offsets [S+1] int32 on the host."""
    cu = np.zeros(len(seqlens) + 1, np.int64)
    cu[1:] = np.cumsum(np.asarray(seqlens, np.int64))
    return torch.from_numpy(cu.astype(np.int32))


def _block_ids(seqlens, block_size: int) -> torch.Tensor:
    """For each token, the index of its block counted over the whole batch
    (blocks restart at every sequence).  Layout bookkeeping for the offsets."""
    ids = []
    base = 0
    for L in seqlens:
        local = torch.arange(L, dtype=torch.int64) // block_size
        ids.append(local + base)
        base += (L + block_size - 1) // block_size
    if not ids:
        return torch.zeros(0, dtype=torch.int64), 0
    return torch.cat(ids), base


def make(seqlens, hq: int, hkv: int, d: int, dtype, block_size: int, key_offset_std: float = 0.0,
         seed: int = 0, device="cpu"):
    """Draw (q, k, v, cu_seqlens).  q [T, hq, d], k/v [T, hkv, d] in `dtype` on
    `device`; cu_seqlens int32 on the host."""
    seqlens = tuple(int(x) for x in seqlens)
    T = sum(seqlens)
    dev = torch.device(device)
    gen = torch.Generator(device=dev)
    gen.manual_seed(int(seed))
    q = torch.randn((T, hq, d), generator=gen, device=dev, dtype=torch.float32)
    k = torch.randn((T, hkv, d), generator=gen, device=dev, dtype=torch.float32)
    v = torch.randn((T, hkv, d), generator=gen, device=dev, dtype=torch.float32)
    if key_offset_std > 0.0 and T > 0:
        ids, nblk = _block_ids(seqlens, block_size)
        off = torch.randn((nblk, hkv, d), generator=gen, device=dev, dtype=torch.float32)
        off.mul_(float(key_offset_std))
        k.add_(off[ids.to(dev)])
        del off
    if dtype != torch.float32:
        q, k, v = q.to(dtype), k.to(dtype), v.to(dtype)
    return q, k, v, cu_seqlens(seqlens)


def make_chunked(seqlens, hq: int, hkv: int, d: int, dtype, block_size: int,
                 key_offset_std: float = 0.0, seed: int = 0, device="cpu",
                 chunk_tokens: int = 1 << 18):
    """Like make(), for prefills too long to draw in fp32 at once: the block
    offsets come first from a generator seeded with `seed`; then the tokens
    are drawn in chunks of chunk_tokens, chunk c from a generator seeded with
    seed * 1000003 + c + 1 (Q, K, V of the chunk in that order, fp32), and
    each chunk is rounded to `dtype` as it is written.  Defines its own
    workloads: the values differ from make() for the same seed."""
    seqlens = tuple(int(x) for x in seqlens)
    T = sum(seqlens)
    dev = torch.device(device)
    q = torch.empty((T, hq, d), device=dev, dtype=dtype)
    k = torch.empty((T, hkv, d), device=dev, dtype=dtype)
    v = torch.empty((T, hkv, d), device=dev, dtype=dtype)
    ids, nblk = _block_ids(seqlens, block_size)
    off = None
    if key_offset_std > 0.0 and T > 0:
        gen = torch.Generator(device=dev)
        gen.manual_seed(int(seed))
        off = torch.randn((nblk, hkv, d), generator=gen, device=dev, dtype=torch.float32)
        off.mul_(float(key_offset_std))
    for c, t0 in enumerate(range(0, T, chunk_tokens)):
        t1 = min(T, t0 + chunk_tokens)
        gen = torch.Generator(device=dev)
        gen.manual_seed(int(seed) * 1000003 + c + 1)
        qc = torch.randn((t1 - t0, hq, d), generator=gen, device=dev, dtype=torch.float32)
        kc = torch.randn((t1 - t0, hkv, d), generator=gen, device=dev, dtype=torch.float32)
        vc = torch.randn((t1 - t0, hkv, d), generator=gen, device=dev, dtype=torch.float32)
        if off is not None:
            kc.add_(off[ids[t0:t1].to(dev)])
        q[t0:t1].copy_(qc)
        k[t0:t1].copy_(kc)
        v[t0:t1].copy_(vc)
        del qc, kc, vc
    return q, k, v, cu_seqlens(seqlens)


def make_dout(shape, dtype, seed: int = 0, device="cpu", chunk_tokens: int = 1 << 18):
    """Upstream gradient dL/d(out) for the backward pass: entries i.i.d.
    N(0, 1), drawn in fp32 in chunks of chunk_tokens rows of `shape` =
    (T, Hq, D), chunk c from a generator seeded with seed * 7919 + c + 17, and
    rounded once to `dtype`."""
    T = int(shape[0])
    dev = torch.device(device)
    out = torch.empty(tuple(shape), device=dev, dtype=dtype)
    for c, t0 in enumerate(range(0, T, chunk_tokens)):
        t1 = min(T, t0 + chunk_tokens)
        gen = torch.Generator(device=dev)
        gen.manual_seed(int(seed) * 7919 + c + 17)
        out[t0:t1].copy_(torch.randn((t1 - t0,) + tuple(shape[1:]), generator=gen, device=dev,
                                     dtype=torch.float32))
    return out


# Sweeps, 32 query / 8 kv heads, D = 128, bf16, key offsets N(0, 0.5^2),
# chunked generation; points are (tokens, block size, top-k):
#   fig2a: 8K .. 1M tokens at block size 4096 and top-12 (the 1M model's
#          setting, Fig. 2a);
#   fig2b: 8K .. 10M tokens with 64 blocks per sequence (B = L / 64) and
#          top-3, a fixed tail sparsity of 1 - 3/64 = 95.31% (Fig. 2b);
#   gran:  32K tokens at a fixed tail sparsity of 75% with finer and finer
#          blocks, (B, k) = (4096, 2) .. (256, 32) (the block-granularity
#          ablation of Sec. 3.1).
SWEEP_POINTS = {
    "fig2a": [(L, 4096, 12) for L in (8192, 16384, 32768, 65536, 131072, 262144, 524288, 1048576)],
    "fig2b": [(L, L // 64, 3) for L in (8192, 32768, 131072, 524288, 1048576, 2097152, 4194304,
                                          8388608, 10485760)],
    "gran": [(32768, 4096, 2), (32768, 2048, 4), (32768, 1024, 8), (32768, 512, 16),
             (32768, 256, 32)],
}


def sweep_workload(kind: str, L: int, B: int = None, k: int = None) -> Workload:
    """The sweep point of `kind` with L tokens (and, for gran, block size B)."""
    pts = SWEEP_POINTS[kind]
    idx = [i for i, (l, b, kk) in enumerate(pts) if l == L and (B is None or b == B)]
    if not idx:
        raise ValueError((kind, L, B))
    i = idx[0]
    L, B, k = pts[i]
    seed = 100 + i + {"fig2a": 0, "fig2b": 50, "gran": 80}[kind]
    return Workload("bf16_L%d_gqa32x8_B%d_k%d_%s" % (L, B, k, kind), (L,), 32, 8, 128, "bf16", B, k,
                    0.5, seed, "sweep %s" % kind)


def sweep_workloads(kind: str):
    return [sweep_workload(kind, L, B) for (L, B, _) in SWEEP_POINTS[kind]]


def make_workload(w: Workload, device="cpu"):
    if w.name.rsplit("_", 1)[-1] in SWEEP_POINTS:
        return make_chunked(w.seqlens, w.hq, w.hkv, w.d, w.torch_dtype, w.block_size,
                            w.key_offset_std, w.seed, device)
    return make(w.seqlens, w.hq, w.hkv, w.d, w.torch_dtype, w.block_size, w.key_offset_std,
                w.seed, device)


def to_oracle(x: torch.Tensor) -> np.ndarray:
    """Host numpy view of an input for the oracle: float32 as is, bf16 as its
    uint16 bit pattern (the oracle widens it exactly)."""
    x = x.detach().contiguous().cpu()
    if x.dtype == torch.float32:
        return x.numpy()
    if x.dtype == torch.bfloat16:
        return x.view(torch.int16).numpy().view(np.uint16)
    raise TypeError(x.dtype)


def sample_rows(w: Workload, n_uniform: int = 64, full_heads=(0, -1), seed: int = 1234):
    """Row ids (t * hq + h) of the sampled-output check at full size: for every
    q-head the block-boundary positions tau in {0, 1, B-1, B, (k-1)B-1, (k-1)B,
    kB-1, kB, L/2, L-B, L-1} of every sequence, n_uniform seeded uniform
    positions, and every row of the last block for the heads in full_heads."""
    B, k = w.block_size, w.topk
    rng = np.random.default_rng(seed)
    rows = set()
    start = 0
    heads_full = {h % w.hq for h in full_heads}
    for L in w.seqlens:
        if L == 0:
            continue
        taus = {0, 1, B - 1, B, (k - 1) * B - 1, (k - 1) * B, k * B - 1, k * B, L // 2, L - B, L - 1}
        taus = {t for t in taus if 0 <= t < L}
        for h in range(w.hq):
            pos = set(taus) | set(int(x) for x in rng.integers(0, L, size=n_uniform))
            if h in heads_full:
                pos |= set(range(((L - 1) // B) * B, L))
            for t in pos:
                rows.add((start + t) * w.hq + h)
        start += L
    return np.array(sorted(rows), dtype=np.int64)
