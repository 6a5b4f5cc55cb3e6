"""Benchmark of the MoBA causal prefill forward on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--dense-steps N] [--no-cpu]
    python bench.py --sweep fig2a|fig2b|gran [--sweep-steps K] [--sweep-lengths L1,L2,..]
    python bench.py --backward [--steps K] [--warmup W] [--workload NAME] [--no-cpu]
    python bench.py --decode [--steps K] [--workload NAME] [--no-cpu]

One step = one moba_forward call over the whole workload (pool, gate, route,
history and current-block attention, merge), inputs resident in HBM.  The
default workload is the 1M-token prefill (32 query heads, 8 kv-heads, head
dim 128, bf16, block 4096, top-12).  Prints one JSON line:
  value          attended TFLOP/s of the whole forward (4*D per attended
                 query-key pair; the causal triangle of the current block plus
                 B keys per selected history block)
  ms_per_step    forward latency
  config         workload, bf16-peak fraction, dense latency and speedup
  roofline       the history-attention kernel (the dominant one): algorithmic
                 FLOPs per launch / its mean launch time from HIP events on
                 the library's stream, against the 2516.6 TFLOP/s bf16 peak
  cpu_baseline   the fp64 oracle on a fixed sample of rows, host cores
--backward and --decode print one line each of their own, with their own
oracle baseline (dQ of sampled rows; the whole decode call); --no-cpu skips
every baseline.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402
import torch  # noqa: E402

from paper_2502_13189_amd import binding, inputs  # noqa: E402

BF16_PEAK_TFLOPS = 2516.6   # 256 CUs x 4096 bf16 FLOP/clk x 2.4 GHz (dense)
HBM_PEAK_GBS = 8000.0

# HBM traffic of the history-attention kernel, measured with rocprofv3 counter
# passes and stored with a hash of the kernel sources it was measured on; it
# is reported only while the sources are unchanged.
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "attn_hist_L1M_gqa32x8_B4096_k12_traffic.md")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2502_13189_amd", "csrc", f)
                  for f in ("attn_mfma.hip", "mfma_tile.h", "moba_internal.h")]


def kernel_source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload):
    """Bytes per history-attention launch from the committed counter profile,
    or None if it is missing, for another workload or for other sources."""
    try:
        text = open(TRAFFIC_PROFILE).read()
    except OSError:
        return None
    fields = {}
    for line in text.splitlines():
        if line.startswith("- ") and ": " in line:
            k, v = line[2:].split(": ", 1)
            fields[k.strip()] = v.strip().strip("`")
    if fields.get("workload") != workload or fields.get("source_sha256") != kernel_source_hash():
        return None
    try:
        return float(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def attended_keys(seqlens, B, topk):
    """(current-block keys, history keys, history selections) per query head."""
    cur = hist = sel = 0
    for L in seqlens:
        n = (L + B - 1) // B
        for c in range(n):
            m = min(L, (c + 1) * B) - c * B
            cur += m * (m + 1) // 2
            h = min(topk - 1, c)
            hist += m * B * h
            sel += m * h
    return cur, hist, sel


def dense_keys(seqlens):
    return sum(L * (L + 1) // 2 for L in seqlens)


def time_steps(fn, steps, warmup):
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / max(steps, 1)


def cpu_baseline(w, q, k, v, cu, n_rows, seed=7):
    """The oracle on n_rows seeded rows of the workload: pool over all keys,
    gate and attention for the sampled rows.  Returns a dict."""
    from oracle import oracle

    cores = len(os.sched_getaffinity(0))
    oracle.set_threads(cores)
    T, Hq = q.shape[0], q.shape[1]
    n_rows = min(n_rows, T * Hq)
    rng = np.random.default_rng(seed)
    rows = np.sort(rng.choice(T * Hq, size=n_rows, replace=False)).astype(np.int64)
    t_copy = time.perf_counter()
    rows_t = torch.as_tensor(rows, device=q.device)
    kn, vn = inputs.to_oracle(k), inputs.to_oracle(v)
    qn = inputs.to_oracle(q)
    t_copy = time.perf_counter() - t_copy
    cun = cu.numpy()
    t0 = time.perf_counter()
    kbar = oracle.pool(kn, cun, w.block_size)
    t1 = time.perf_counter()
    sel = oracle.select(qn, kbar, cun, w.block_size, w.topk, rows=rows)
    _, _ = oracle.attend(qn, kn, vn, cun, w.block_size, sel, rows=rows)
    t2 = time.perf_counter()
    # attended keys of the sampled rows
    cum = np.asarray(cun, np.int64)
    t = rows // Hq
    s = np.searchsorted(cum, t, side="right") - 1
    tau = t - cum[s]
    c = tau // w.block_size
    keys = (tau - c * w.block_size + 1) + w.block_size * np.minimum(w.topk - 1, c)
    flop = 4.0 * w.d * float(keys.sum())
    del rows_t
    return {
        "value": flop / (t2 - t1) / 1e12,
        "unit": "TFLOP/s",
        "cores": oracle.threads(),
        "kind": "oracle",
        "sample": ("fp64 oracle gate + attention for %d seeded rows (t*Hq+h) of the %s workload "
                   "(%.3g attended FLOP) in %.1f s; its block mean-pool over all keys took %.1f s "
                   "and is not in the rate; host copy %.1f s" %
                   (n_rows, w.name, flop, t2 - t1, t1 - t0, t_copy)),
        "cpu_model": _cpu_model(),
    }


def cpu_baseline_backward(w, q, k, v, dout, cu, n_rows, seed=7):
    """The oracle's backward on n_rows seeded rows of the workload: the
    query-side gradient dQ (the S, dP and dQ products, 6*D FLOP per attended
    pair, for the oracle's own selection of those rows).  The key-side
    gradients would need fp64 accumulators over every key and are left out."""
    from oracle import oracle

    oracle.set_threads(len(os.sched_getaffinity(0)))
    T, Hq, D = q.shape
    rng = np.random.default_rng(seed)
    rows = np.sort(rng.choice(T * Hq, size=n_rows, replace=False)).astype(np.int64)
    rows_t = torch.as_tensor(rows, device=q.device)
    q_r = inputs.to_oracle(q.reshape(T * Hq, D)[rows_t])
    d_r = inputs.to_oracle(dout.reshape(T * Hq, D)[rows_t])
    kn, vn = inputs.to_oracle(k), inputs.to_oracle(v)
    cun = cu.numpy()
    kbar = oracle.pool(kn, cun, w.block_size)
    sel = oracle.select_rows(q_r, T, Hq, kbar, cun, w.block_size, w.topk, rows)
    t0 = time.perf_counter()
    oracle.attend_backward(q_r, kn, vn, d_r, cun, w.block_size, sel, rows=rows, shape=(T, Hq))
    t1 = time.perf_counter()
    cum = np.asarray(cun, np.int64)
    t = rows // Hq
    s = np.searchsorted(cum, t, side="right") - 1
    tau = t - cum[s]
    c = tau // w.block_size
    keys = (tau - c * w.block_size + 1) + w.block_size * np.minimum(w.topk - 1, c)
    flop = 6.0 * D * float(keys.sum())
    return {
        "value": flop / (t1 - t0) / 1e12,
        "unit": "TFLOP/s",
        "cores": oracle.threads(),
        "kind": "oracle",
        "sample": ("fp64 oracle dQ (S, dP, dQ: 6*D FLOP per attended pair) of %d seeded rows "
                   "(t*Hq+h) of the %s workload for the oracle's selection: %.3g FLOP in %.1f s"
                   % (n_rows, w.name, flop, t1 - t0)),
        "cpu_model": _cpu_model(),
    }


def cpu_baseline_decode(w, qd, k, v, cu):
    """The oracle on the decode workload itself (every sequence's new query,
    every head): full attention over the cache, and MoBA (block means of the
    cache, gate, attention).  Milliseconds per decode call."""
    from oracle import oracle

    oracle.set_threads(len(os.sched_getaffinity(0)))
    S, Hq, D = qd.shape
    T = int(cu[-1])
    q_rows = inputs.to_oracle(qd.reshape(S * Hq, D))
    kn, vn = inputs.to_oracle(k), inputs.to_oracle(v)
    cun = cu.numpy()
    rows = np.array([(int(cun[s + 1]) - 1) * Hq + h for s in range(S) for h in range(Hq)], np.int64)
    t0 = time.perf_counter()
    oracle.attend_rows(q_rows, T, Hq, kn, vn, cun, max(w.seqlens), np.zeros((len(rows), 1), np.int32),
                       rows)
    t1 = time.perf_counter()
    kbar = oracle.pool(kn, cun, w.block_size)
    sel = oracle.select_rows(q_rows, T, Hq, kbar, cun, w.block_size, w.topk, rows)
    oracle.attend_rows(q_rows, T, Hq, kn, vn, cun, w.block_size, sel, rows)
    t2 = time.perf_counter()
    return {
        "value": {"full": round((t1 - t0) * 1e3, 1), "moba": round((t2 - t1) * 1e3, 1)},
        "unit": "ms per decode call",
        "cores": oracle.threads(),
        "kind": "oracle",
        "sample": ("the whole decode call (%d rows) in fp64: full attention over the cache; MoBA "
                   "with the block mean-pool of the cache included" % len(rows)),
        "cpu_model": _cpu_model(),
    }


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def run_sweep(args):
    """A sweep (Fig. 2a or 2b lengths, or the block-granularity points): one
    JSON line per point with the forward time, attended TFLOP/s and, up to
    --sweep-dense-max tokens, the dense causal time and measured speedup;
    beyond it the dense time is extrapolated at the rate of the largest
    measured dense point and labelled as such."""
    dev = torch.device("cuda:0")
    points = inputs.sweep_workloads(args.sweep)
    if args.sweep_lengths:
        keep = {int(x) for x in args.sweep_lengths.split(",")}
        points = [w for w in points if w.seqlens[0] in keep]
    dense_rate = None  # FLOP per ms of the largest measured dense point
    for w in points:
        L = w.seqlens[0]
        print("[bench] sweep %s %s" % (args.sweep, w.name), file=sys.stderr, flush=True)
        q, k, v, cu = inputs.make_workload(w, device=dev)
        out = torch.empty_like(q)
        lse = torch.empty((w.hq, L), dtype=torch.float32, device=dev)
        step = lambda: binding.forward(q, k, v, cu, w.block_size, w.topk, out=out, lse=lse)
        if L < (1 << 22):
            ms = time_steps(step, args.sweep_steps, 1)
            # one more step with per-phase events (not in the timing)
            binding.profile_read()
            binding.profile_enable(True)
            step()
            torch.cuda.synchronize()
            binding.profile_enable(False)
            phases = binding.profile_read()
        else:
            # steps of many seconds: the events of the timed steps give the
            # phases (their cost is negligible at this scale), no warm-up
            binding.profile_read()
            binding.profile_enable(True)
            ms = time_steps(step, args.sweep_steps, 0)
            binding.profile_enable(False)
            phases = {n: (c, t / args.sweep_steps) for n, (c, t) in binding.profile_read().items()}
        cur, hist, _ = attended_keys(w.seqlens, w.block_size, w.topk)
        flop = 4.0 * w.d * w.hq * (cur + hist)
        dflop = 4.0 * w.d * w.hq * dense_keys(w.seqlens)
        dense_ms, dense_kind = None, None
        if L <= args.sweep_dense_max:
            dense_ms = time_steps(lambda: binding.dense_forward(q, k, v, cu, out=out, lse=lse), 1,
                                  1 if L <= 262144 else 0)
            dense_kind = "measured"
            dense_rate = dflop / dense_ms
        elif dense_rate:
            dense_ms = dflop / dense_rate
            dense_kind = "extrapolated at the largest measured dense rate"
        tflops = flop / (ms * 1e-3) / 1e12
        print(json.dumps({
            "sweep": args.sweep, "workload": w.name, "tokens": L, "block_size": w.block_size,
            "topk": w.topk, "q_heads": w.hq, "kv_heads": w.hkv, "steps": args.sweep_steps,
            "ms": round(ms, 3), "attended_flop": flop, "tflops": round(tflops, 2),
            "pct_bf16_peak": round(100.0 * tflops / BF16_PEAK_TFLOPS, 2),
            "dense_flop": dflop, "flop_ratio": round(dflop / flop, 3),
            "dense_ms": None if dense_ms is None else round(dense_ms, 2), "dense": dense_kind,
            "speedup_vs_dense": None if dense_ms is None else round(dense_ms / ms, 3),
            "phases_ms": {n: round(t, 3) for n, (c, t) in phases.items()},
        }), flush=True)
        del q, k, v, out, lse
        torch.cuda.empty_cache()


def run_backward(args):
    """The backward pass (moba_backward) on the workload: one JSON line with
    its time and rates.  Algorithmic FLOPs count the five products of the
    attention backward (S recomputed, dP, dV, dK, dQ: 10*D per attended
    query-key pair, 2.5x the forward's); the kernels execute seven (S and dP
    are computed on both the query and the key side)."""
    w = inputs.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    print("[bench] generating %s" % w.name, file=sys.stderr, flush=True)
    q, k, v, cu = inputs.make_workload(w, device=dev)
    dout = inputs.make_dout(q.shape, q.dtype, w.seed, device=dev)
    out, lse = binding.forward(q, k, v, cu, w.block_size, w.topk)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    torch.cuda.synchronize()

    def step():
        binding.backward(q, k, v, cu, w.block_size, w.topk, out, lse, dout, dq=dq, dk=dk, dv=dv)

    print("[bench] backward warmup %d" % args.warmup, file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print("[bench] backward timing %d steps" % args.steps, file=sys.stderr, flush=True)
    binding.profile_read()
    binding.profile_enable(True)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    binding.profile_enable(False)
    phases = binding.profile_read()
    cur, hist, _ = attended_keys(w.seqlens, w.block_size, w.topk)
    pairs = w.hq * (cur + hist)
    flop = 10.0 * w.d * pairs
    tflops = flop / (ms * 1e-3) / 1e12

    def kernel_rate(name, kflop):
        """Executed TFLOP/s of a phase: kflop per step over its time per step."""
        n, t = phases.get(name, (0, 0.0))
        return None if not n else round(kflop / (t / args.steps * 1e-3) / 1e12, 2)

    # executed products per kernel: dq history 3 (S, dP, dQ) over history
    # pairs; dq current 3 over current-block pairs; dkdv 4 (S, dP, dV, dK)
    # over all pairs
    rates = {
        "bwd_dq_hist": kernel_rate("bwd_dq_hist", 6.0 * w.d * w.hq * hist),
        "bwd_dq_cur": kernel_rate("bwd_dq_cur", 6.0 * w.d * w.hq * cur),
        "bwd_dkdv": kernel_rate("bwd_dkdv", 8.0 * w.d * pairs),
    }
    cpu = None
    if not args.no_cpu:
        n_rows = max(1, args.cpu_rows * 2 // 3)
        print("[bench] oracle baseline: dQ of %d rows" % n_rows, file=sys.stderr, flush=True)
        cpu = cpu_baseline_backward(w, q, k, v, dout, cu, n_rows)
    print(json.dumps({
        "mode": "backward", "workload": w.name, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 3), "algorithmic_flop": flop, "tflops": round(tflops, 2),
        "pct_bf16_peak": round(100.0 * tflops / BF16_PEAK_TFLOPS, 2), "dtype": "bf16",
        "data": "synthetic",
        "phases_ms_per_step": {n: round(t / args.steps, 3) for n, (c, t) in phases.items()},
        "executed_tflops_per_kernel": rates,
        "cpu_baseline": cpu,
    }), flush=True)


def run_decode(args):
    """Decode on the workload's cache: one new query per sequence (the last
    token's), full attention (the paper's choice for generation) and MoBA
    with the cache's block means kept by the caller.  One JSON line with both
    latencies and their HBM rates: bytes = the K/V rows each mode must read
    (full: every cached key of every kv-head; MoBA: the union of the blocks
    the group's query heads select, from the prefill gate's selection of the
    same rows) plus the queries, block means and outputs."""
    w = inputs.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    print("[bench] generating %s" % w.name, file=sys.stderr, flush=True)
    q, k, v, cu = inputs.make_workload(w, device=dev)
    last = (cu[1:] - 1).to(torch.int64).to(dev)
    qd = q[last].contiguous()
    S, Hq, Hkv, D, B = len(w.seqlens), w.hq, w.hkv, w.d, w.block_size
    G = Hq // Hkv
    kbar = binding.pool(k, cu, B)
    sel = binding.select(q, k, cu, B, w.topk)[last].cpu().numpy()  # [S, Hq, topk]
    del q
    torch.cuda.synchronize()
    out = torch.empty_like(qd)
    lse = torch.empty((Hq, S), dtype=torch.float32, device=dev)
    res = {}
    for mode, kk in (("full", 0), ("moba", w.topk)):
        step = lambda: binding.decode(qd, k, v, cu, B, kk, kbar=kbar, out=out, lse=lse)
        for _ in range(max(args.warmup, 1)):
            step()
        torch.cuda.synchronize()
        binding.profile_read()
        binding.profile_enable(True)
        t0 = time.perf_counter()
        n = max(args.steps, 1) * 20
        for _ in range(n):
            step()
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / n
        binding.profile_enable(False)
        phases = binding.profile_read()
        if mode == "full":
            kv_rows = sum(w.seqlens) * Hkv
        else:
            kv_rows = 0
            for s_, L in enumerate(w.seqlens):
                for g in range(Hkv):
                    blocks = set(int(j) for j in sel[s_, g * G:(g + 1) * G].ravel() if j >= 0)
                    kv_rows += sum(min(B, L - j * B) for j in blocks)
        nbytes = kv_rows * 2 * D * 2 + S * Hq * D * 2 * 2 + (kbar.numel() * 4 if mode == "moba" else 0)
        res[mode] = {"ms": round(ms, 4), "kv_rows_read": kv_rows, "bytes": nbytes,
                     "gb_per_s": round(nbytes / (ms * 1e-3) / 1e9, 1),
                     "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "phases_ms": {k_: round(t / c, 4) for k_, (c, t) in phases.items()}}
    cpu = None
    if not args.no_cpu:
        print("[bench] oracle baseline: both decode modes", file=sys.stderr, flush=True)
        cpu = cpu_baseline_decode(w, qd, k, v, cu)
    print(json.dumps({"mode": "decode", "workload": w.name, "queries": S * Hq, "dtype": "bf16",
                      "data": "synthetic", "full": res["full"], "moba": res["moba"],
                      "speedup_moba_vs_full": round(res["full"]["ms"] / res["moba"]["ms"], 3),
                      "cpu_baseline": cpu}),
          flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default=inputs.HEADLINE, choices=sorted(inputs.WORKLOADS))
    ap.add_argument("--dense-steps", type=int, default=1)
    ap.add_argument("--cpu-rows", type=int, default=12000)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--sweep", choices=sorted(inputs.SWEEP_POINTS),
                    help="length-scaling sweep instead of the headline line (one JSON line "
                         "per length)")
    ap.add_argument("--sweep-steps", type=int, default=2)
    ap.add_argument("--sweep-lengths", default=None, help="comma-separated subset of lengths")
    ap.add_argument("--sweep-dense-max", type=int, default=1 << 20)
    ap.add_argument("--backward", action="store_true",
                    help="time moba_backward on the workload instead (one JSON line)")
    ap.add_argument("--decode", action="store_true",
                    help="time moba_decode (full and MoBA) on the workload's cache instead")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)

    binding.load()
    if args.sweep:
        run_sweep(args)
        return
    if args.backward:
        run_backward(args)
        return
    if args.decode:
        run_decode(args)
        return
    w = inputs.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    print("[bench] generating %s" % w.name, file=sys.stderr, flush=True)
    q, k, v, cu = inputs.make_workload(w, device=dev)
    torch.cuda.synchronize()
    out = torch.empty_like(q)
    lse = torch.empty((w.hq, q.shape[0]), dtype=torch.float32, device=dev)

    def step():
        binding.forward(q, k, v, cu, w.block_size, w.topk, out=out, lse=lse)

    print("[bench] warmup %d" % args.warmup, file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print("[bench] timing %d steps" % args.steps, file=sys.stderr, flush=True)
    binding.profile_read()
    binding.profile_enable(True)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    binding.profile_enable(False)
    phases = binding.profile_read()

    cur, hist, nsel = attended_keys(w.seqlens, w.block_size, w.topk)
    flop = 4.0 * w.d * w.hq * (cur + hist)
    tflops = flop / (ms * 1e-3) / 1e12
    hist_flop_step = 4.0 * w.d * w.hq * hist
    hl, hms = phases.get("attn_hist", (0, 0.0))
    launches_per_step = hl / max(args.steps, 1)
    achieved = (hist_flop_step / launches_per_step) / (hms / hl * 1e-3) / 1e12 if hl else 0.0

    dense_ms = None
    if args.dense_steps > 0:
        print("[bench] dense x%d" % args.dense_steps, file=sys.stderr, flush=True)
        dout = torch.empty_like(q)
        dlse = torch.empty_like(lse)
        dense_ms = time_steps(lambda: binding.dense_forward(q, k, v, cu, out=dout, lse=dlse),
                              args.dense_steps, 1)
        del dout, dlse
    dflop = 4.0 * w.d * w.hq * dense_keys(w.seqlens)

    cpu = None
    if not args.no_cpu:
        print("[bench] oracle baseline on %d rows" % args.cpu_rows, file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, q, k, v, cu, args.cpu_rows)

    res = {
        "metric": "MoBA prefill ms + attended TFLOP/s (% bf16 MFMA peak) at 1M ctx; speedup vs dense",
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "seqlens": list(w.seqlens),
            "q_heads": w.hq, "kv_heads": w.hkv, "head_dim": w.d,
            "block_size": w.block_size, "topk": w.topk,
            "attended_flop": flop,
            "pct_bf16_peak": round(100.0 * tflops / BF16_PEAK_TFLOPS, 2),
            "dense_ms": None if dense_ms is None else round(dense_ms, 2),
            "dense_flop": dflop,
            "dense_tflops": None if dense_ms is None else round(dflop / (dense_ms * 1e-3) / 1e12, 2),
            "speedup_vs_dense": None if dense_ms is None else round(dense_ms / ms, 3),
            "phases_ms_per_step": {n: round(t / args.steps, 3) for n, (c, t) in phases.items()},
        },
        "roofline": {
            "kernel": "attn_mfma_kernel<history> (history-block attention)",
            "bound": "mfma",
            "achieved": round(achieved, 2),
            "peak": BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / BF16_PEAK_TFLOPS, 4),
            "traffic": measured_traffic(w.name),
            "flop_per_launch": hist_flop_step / max(launches_per_step, 1),
            "launches_per_step": launches_per_step,
            "mean_launch_ms": round(hms / hl, 3) if hl else None,
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
