/*
 * moba.h -- C ABI of the MI355X (gfx950) MoBA causal prefill library.
 *
 * MoBA (Mixture of Block Attention, arXiv 2502.13189) lets every query attend
 * to its own block plus the top-scoring past blocks of its sequence.  The
 * library computes, on one GPU:
 *   block mean-pool of the keys  -> gate (unscaled q . block key, causal mask,
 *   forced current block, top-k)  -> routing inversion (queries per block)
 *   -> attention over the routed history blocks and the causal current block
 *   -> log-sum-exp merge of the partial results,
 * following Sec. 2.2 (Eq. 2-6) and Algorithm 1 of the paper; plus dense causal
 * attention (Eq. 1) built from the same kernels, for comparison.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Tensors are passed as moba_tensor descriptors: a data pointer, a dtype, and
 * shape/stride in ELEMENTS.  The caller owns every tensor; the library never
 * frees caller memory.  All tensors except cu_seqlens live in device memory of
 * the current HIP device.
 *
 *   q    [T, Hq,  D]  bf16 or f32; last dim contiguous, any token/head stride
 *   k, v [T, Hkv, D]  same dtype as q; last dim contiguous
 *   out  [T, Hq,  D]  same dtype as q; last dim contiguous
 *   lse  [Hq, T]      f32, contiguous; natural-log log-sum-exp of the scaled
 *                      logits over the keys each query attended
 *   cu_seqlens [S+1]  int32, contiguous, host OR device memory: cu[0] = 0,
 *                      non-decreasing, cu[S] = T.  Sequence s holds tokens
 *                      [cu[s], cu[s+1]); blocks restart at every sequence and
 *                      nothing is attended across sequences.  A device
 *                      cu_seqlens is copied to the host on `stream` (after
 *                      the work enqueued there before the call) and the
 *                      stream is waited for; pass it in host memory to keep
 *                      the call asynchronous.
 *
 * Head dimension D must be 128.  Hq must be a multiple of Hkv (GQA: query head
 * h uses kv-head h / (Hq / Hkv)) and Hq / Hkv <= 128.  Logits are scaled by
 * 1/sqrt(D); gate scores are not scaled (Eq. 6).
 *
 * Every call enqueues its device work on `stream` and returns without waiting,
 * except as noted.  Arguments are validated before any HIP call; invalid
 * arguments return a status code and touch nothing.  Kernel launch failures
 * return MOBA_ERR_HIP.  No function throws.
 *
 * Per-shape tables (sequence offsets, tile lists) are built on the host for
 * each new (cu_seqlens, heads, block size, top-k) and copied on `stream`; the
 * last few are kept per device.  Their buffers grow in powers of two, and
 * growing one synchronizes the device.
 *
 * The library keeps one cached device workspace per device, grown on demand
 * (growing it synchronizes the device) and capped by the environment variable
 * MOBA_WORKSPACE_LIMIT_BYTES (default 64 GiB).  When one call needs more, the
 * attention runs in chunks of kv-heads.  The workspace is shared by all calls
 * on a device: calls on one device must come from one host thread, and calls
 * enqueued on different streams of one device must not overlap in time.
 */
#ifndef MOBA_H_
#define MOBA_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { MOBA_F32 = 0, MOBA_BF16 = 1, MOBA_I32 = 2, MOBA_I64 = 3 } moba_dtype;

typedef struct {
  void* data;        /* host or device pointer, see each argument */
  int32_t dtype;     /* moba_dtype */
  int32_t ndim;      /* 1..4 */
  int64_t shape[4];  /* elements per dimension */
  int64_t stride[4]; /* elements between consecutive indices of a dimension */
} moba_tensor;

typedef enum {
  MOBA_OK = 0,
  MOBA_ERR_NULL = 1,        /* a required descriptor or data pointer is NULL */
  MOBA_ERR_DTYPE = 2,       /* dtype mismatch or unsupported dtype */
  MOBA_ERR_SHAPE = 3,       /* shapes disagree with each other or with cu_seqlens */
  MOBA_ERR_LAYOUT = 4,      /* last dim not contiguous, or a contiguous tensor required */
  MOBA_ERR_BLOCK_SIZE = 5,  /* block_size < 1 */
  MOBA_ERR_TOPK = 6,        /* topk < 1 */
  MOBA_ERR_SEQLENS = 7,     /* cu[0] != 0, decreasing, or cu[S] != T */
  MOBA_ERR_UNSUPPORTED = 8, /* D != 128, Hq/Hkv > 128, > 4096 blocks per sequence,
                               1 < topk-1 < #blocks with topk > 64, or index overflow */
  MOBA_ERR_NO_MEMORY = 9,   /* workspace over MOBA_WORKSPACE_LIMIT_BYTES or hipMalloc failed */
  MOBA_ERR_HIP = 10         /* a HIP call or kernel launch failed */
} moba_status;

/*
 * MoBA causal prefill forward (Sec. 2.2 Eq. 2-6; Algorithm 1).
 *
 * For query token t of sequence s at local position tau = t - cu[s] and
 * query head h: c = tau / block_size is its current block.  The gate scores
 * every past block j < c with <q, mean of block j's keys> (unscaled, fp32),
 * keeps the min(topk-1, c) highest (equal scores: lower block index wins),
 * and adds block c (the current block counts toward topk).  out[t, h] is
 * softmax attention over every key of the kept past blocks plus the keys of
 * block c up to and including t.  lse[h, t] is its log-sum-exp.
 * topk larger than the number of blocks selects every causal block: when
 * topk is at least the block count of the longest sequence, every row
 * attends its whole causal prefix and the call runs moba_dense_forward's
 * kernels (the same result up to rounding).
 *
 * Arguments: see the conventions above.  block_size >= 1, topk >= 1.
 * Returns MOBA_OK or an error status; on error nothing has been enqueued
 * unless the status is MOBA_ERR_HIP.
 */
moba_status moba_forward(const moba_tensor* q, const moba_tensor* k, const moba_tensor* v,
                         const moba_tensor* cu_seqlens, int32_t block_size, int32_t topk,
                         moba_tensor* out, moba_tensor* lse, hipStream_t stream);

/*
 * MoBA backward: gradients of moba_forward's output w.r.t. q, k and v.  The
 * gate (Eq. 3 and Eq. 5) is a hard 0/1 choice and passes no gradient, so
 * these are the gradients of softmax attention (Eq. 2) over the key set of
 * Eq. 4 that the forward selected.
 *
 * q, k, v, cu_seqlens, block_size, topk: exactly as passed to moba_forward;
 *   the selection is recomputed from them and equals the forward's.
 * out [T, Hq, D], lse [Hq, T]: moba_forward's results for these inputs.
 * dout [T, Hq, D]: gradient of the loss w.r.t. out.
 * dq [T, Hq, D], dk, dv [T, Hkv, D]: outputs, overwritten; dk and dv of a
 *   kv-head sum over the query heads of its group.
 * bf16 only: f32 inputs return MOBA_ERR_DTYPE.  Layout rules as for
 * moba_forward (last dim contiguous, 16-byte aligned rows, any token/head
 * stride).  Products accumulate in fp32; the softmax weights P and the score
 * gradients dS are rounded to bf16 for the second matrix-core products;
 * Delta = <dout, out> per row uses the bf16 out.  Deterministic: no atomics,
 * fixed summation order.  When topk is at least the block count of the
 * longest sequence, this is moba_dense_backward, as in moba_forward.
 */
moba_status moba_backward(const moba_tensor* q, const moba_tensor* k, const moba_tensor* v,
                          const moba_tensor* cu_seqlens, int32_t block_size, int32_t topk,
                          const moba_tensor* out, const moba_tensor* lse, const moba_tensor* dout,
                          moba_tensor* dq, moba_tensor* dk, moba_tensor* dv, hipStream_t stream);

/*
 * Dense causal attention (Eq. 1 with a causal mask and scale 1/sqrt(D)):
 * every query attends to every key of its sequence up to and including
 * itself.  Same tensor conventions as moba_forward.
 */
moba_status moba_dense_forward(const moba_tensor* q, const moba_tensor* k, const moba_tensor* v,
                               const moba_tensor* cu_seqlens, moba_tensor* out, moba_tensor* lse,
                               hipStream_t stream);

/*
 * Backward of moba_dense_forward: gradients of causal full attention (Eq. 1)
 * w.r.t. q, k and v, with out and lse from moba_dense_forward.  Same
 * conventions, dtype (bf16 only) and precision as moba_backward.  With
 * moba_dense_forward it lets a caller switch any attention call between
 * full attention and MoBA, in both directions (the per-layer choice of
 * Sec. 2.2 "Hybrid of MoBA and Full Attention" and the layer-wise hybrid of
 * Sec. 3.2, whose last layers stay full attention).
 */
moba_status moba_dense_backward(const moba_tensor* q, const moba_tensor* k, const moba_tensor* v,
                                const moba_tensor* cu_seqlens, const moba_tensor* out,
                                const moba_tensor* lse, const moba_tensor* dout, moba_tensor* dq,
                                moba_tensor* dk, moba_tensor* dv, hipStream_t stream);

/*
 * Decode: one new query per sequence against its key/value cache.
 *
 * q [S, Hq, D] bf16: the new token of each sequence.  k_cache, v_cache
 * [T, Hkv, D] bf16 hold every sequence's cached keys and values, packed as
 * described by cu_seqlens [S+1] (int32, host or device; every sequence
 * non-empty), and already include each new token's key and value as its
 * sequence's last entry.  So query s sits at position L_s - 1 of sequence s
 * and its result is the last row of the prefill over the cache:
 *   topk >= 1: MoBA with block_size and topk (the gate of Eq. 5 / Eq. 6 over
 *              the sequence's complete past blocks, top-k with the current
 *              block counted, attention over the selected blocks and the
 *              current block up to the query); a topk of at least the
 *              longest sequence's block count selects everything and runs
 *              as topk == 0;
 *   topk == 0: causal full attention over the whole cache (Eq. 1), which is
 *              what the paper uses for generation (Sec. 3.3); block_size is
 *              then ignored.
 * kbar (nullable, MoBA only): the cache's block means as written by
 * moba_pool for the same cu_seqlens and block_size; when NULL they are
 * computed on the fly, which reads the whole key cache.  A decode loop keeps
 * kbar and recomputes it only when a block completes.
 * out [S, Hq, D] bf16 and lse [Hq, S] f32 (natural log) as for moba_forward.
 * Hq / Hkv must not exceed 16.  Gate scores are fp32 sums in a fixed order
 * (four sequential 32-dim partial sums, added in order); near-ties may be
 * broken differently from moba_select's matrix-core gate.  A call whose cu_seqlens differs from those of recent calls (every
 * step of a growing cache) builds new per-shape tables on the host and copies
 * them on `stream`; it does not synchronize the device.
 */
moba_status moba_decode(const moba_tensor* q, const moba_tensor* k_cache,
                        const moba_tensor* v_cache, const moba_tensor* cu_seqlens,
                        const moba_tensor* kbar, int32_t block_size, int32_t topk, moba_tensor* out,
                        moba_tensor* lse, hipStream_t stream);

/*
 * moba_decode without any allocation, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, and
 * harnesses that forbid hipMalloc.  Same arguments, conventions and results
 * as moba_decode (the same kernels; the outputs are bit-identical), except:
 *   - cu_seqlens must be in host memory (a device pointer returns
 *     MOBA_ERR_UNSUPPORTED);
 *   - every intermediate buffer (the per-sequence table, block means when
 *     kbar is NULL, selections, block lists, partial results) lives in one
 *     static device array of MOBA_DECODE_NOALLOC_MAX_BYTES bytes, which each
 *     GPU the library runs on holds from module load until the process ends;
 *     a call needing more returns MOBA_ERR_NO_MEMORY before enqueueing
 *     anything (full attention needs about S * Hq * ceil(L_max / 256) * 516
 *     bytes: a 1M-token cache with 32 query heads fits for one sequence);
 *   - no library call allocates memory, device or pinned, and no profiling
 *     events are recorded.
 * All calls on one GPU share that array and the last call's contents stay
 * in it: calls whose execution overlaps on one GPU (different streams, or
 * host threads) race and give wrong results.  Calls on one stream are
 * ordered and safe.
 */
#define MOBA_DECODE_NOALLOC_MAX_BYTES ((size_t)96 << 20)
moba_status moba_decode_noalloc(const moba_tensor* q, const moba_tensor* k_cache,
                                const moba_tensor* v_cache, const moba_tensor* cu_seqlens,
                                const moba_tensor* kbar, int32_t block_size, int32_t topk,
                                moba_tensor* out, moba_tensor* lse, hipStream_t stream);

/*
 * Block mean-pool of the keys (Eq. 6; Algorithm 1, mean_pool).
 * kbar [nblk_total, Hkv, D] f32 contiguous, device: row b = blk_off[s] + j
 * holds the mean of k over the tokens of block j of sequence s (a short last
 * block uses its own token count), with blk_off[s] = sum over s' < s of
 * ceil(len_s' / block_size).  Accumulated in fp64, rounded once to f32.
 */
moba_status moba_pool(const moba_tensor* k, const moba_tensor* cu_seqlens, int32_t block_size,
                      moba_tensor* kbar, hipStream_t stream);

/*
 * Gate and top-k selection (Eq. 5 and Eq. 6 with the causal rules of
 * Sec. 2.2), including the pool.
 * sel [T, Hq, topk] int32 contiguous, device: the kept past blocks in
 * ascending order, then the current block c, then -1 padding; local block
 * indices of the query's sequence.
 * scores (nullable) [T, Hq, nmax] f32 contiguous, device: the fp32 gate score
 * of every past block j < min(c, nmax), NaN elsewhere (a debugging aid; costs
 * one extra write pass).
 */
moba_status moba_select(const moba_tensor* q, const moba_tensor* k, const moba_tensor* cu_seqlens,
                        int32_t block_size, int32_t topk, moba_tensor* sel, moba_tensor* scores,
                        hipStream_t stream);

/*
 * Routing inversion (Algorithm 1, index_select_moba_attn_block; Sec. 2.3
 * "arrange the ordering of query tokens based on their assigned KV blocks"):
 * for every bin (kv-head g, global block b = blk_off[s] + j) the list of
 * history selections that chose it, by a stable counting sort.
 *   sel      [T, Hq, topk] int32 contiguous, device (as written by moba_select)
 *   counts   [Hkv * nblk_total] int32 contiguous, device: entries per bin,
 *            bins ordered g-major
 *   offsets  [Hkv * nblk_total + 1] int64 contiguous, device: exclusive scan
 *   entries  [E] int32 contiguous, device, E = offsets[last]: entry value
 *            e = r * (topk - 1) + x, where x is the selection slot (position
 *            in sel) and r = g * (T * G) + t * G + (h - g * G) with G = Hq/Hkv;
 *            ascending within a bin.  E must equal the number of history
 *            selections, sum over rows of min(topk - 1, c) (moba_route_size
 *            reports it).
 * num_kv_heads gives Hkv.  The current block is not routed.  A history slot
 * (x < min(topk - 1, c)) whose value is not a past block (outside [0, c)) is
 * skipped, by the counts and the entries alike, so no access leaves the
 * row's bins; offsets[last] then falls short of E and the rest of entries is
 * left unwritten.  moba_select never writes such a slot.
 */
moba_status moba_route(const moba_tensor* sel, const moba_tensor* cu_seqlens, int32_t block_size,
                       int32_t num_kv_heads, moba_tensor* counts, moba_tensor* offsets,
                       moba_tensor* entries, hipStream_t stream);

/*
 * Workspace sizing query: the device workspace bytes moba_forward needs to
 * run in one pass (no kv-head chunking) for any batch of T tokens in
 * nblk_total blocks (sum over sequences of ceil(len / block_size)), with
 * Hq / Hkv heads, head dimension D and topk, for either input dtype.  It is
 * an upper bound over every cu_seqlens with these totals; moba_dense_forward,
 * moba_select and moba_route need no more.  With MOBA_WORKSPACE_LIMIT_BYTES
 * below it the forward runs in more kv-head chunks instead.  The backward
 * needs more (fp32 dQ partials).  Returns 0 for invalid or empty arguments
 * (T < 0, Hq or Hkv < 1, Hq % Hkv != 0, Hq / Hkv > 128, D != 128,
 * topk < 1; T == 0 or nblk_total == 0).  Host-only arithmetic: no HIP call.
 */
size_t moba_workspace_bytes(int64_t T, int32_t Hq, int32_t Hkv, int32_t D, int64_t nblk_total,
                            int32_t topk);

/* Bytes of device workspace the library currently holds on the current device. */
size_t moba_workspace_held_bytes(void);

/*
 * Sizes of moba_route's outputs for a batch (Algorithm 1,
 * index_select_moba_attn_block):
 *   *nblk_total = sum over sequences of ceil(len / block_size), so counts has
 *                 Hkv * *nblk_total entries and offsets one more;
 *   *entries    = E, the number of history selections: num_q_heads times the
 *                 sum over tokens of min(topk - 1, c), c the token's block
 *                 (Eq. 5 keeps min(topk - 1, c) past blocks besides the
 *                 current one; Sec. 3.1 footnote).
 * cu_seqlens as for moba_forward (host or device; a device copy is read on
 * `stream`, which is then waited for).  Errors: MOBA_ERR_NULL,
 * MOBA_ERR_SEQLENS, MOBA_ERR_BLOCK_SIZE, MOBA_ERR_TOPK, MOBA_ERR_SHAPE
 * (num_q_heads < 1).  No device work besides that copy.
 */
moba_status moba_route_size(const moba_tensor* cu_seqlens, int32_t block_size, int32_t topk,
                            int32_t num_q_heads, int64_t* nblk_total, int64_t* entries,
                            hipStream_t stream);

/*
 * The dK/dV kernel of moba_backward hands each 32-row subtile's softmax
 * weights from one wave to another through a flag, with a bounded wait (so
 * that the kernel always ends).  A wait that gives up leaves that subtile's
 * dK wrong; every give-up is counted on the device.  This call waits for the
 * current device, stores the count since the last call in *count and resets
 * it.  With MOBA_DEBUG_SYNC set (non-zero), moba_backward checks the count
 * itself and returns MOBA_ERR_HIP if it is not zero.  Testing aid: with
 * MOBA_FORCE_WAIT_TIMEOUT set (non-zero) every such wait gives up after a
 * few polls.
 */
moba_status moba_take_wait_timeouts(uint64_t* count);

/* Free the cached workspace, tables and counters of the current device
 * (synchronizes the device). */
moba_status moba_release_workspace(void);

/* Static, human-readable name of a status. */
const char* moba_status_string(moba_status status);

/*
 * Per-phase timing.  While enabled, every entry point records HIP events
 * around each phase on the caller's stream.  moba_profile_read waits for the
 * recorded events, writes up to max_phases entries and resets the counters;
 * it returns the number of phases written.
 */
typedef struct {
  char name[24];     /* "pool", "vt_pack", "gate", "route", "attn_hist", ... */
  int64_t launches;  /* phase executions recorded */
  double total_ms;   /* summed event-to-event time */
} moba_phase_stat;

void moba_profile_enable(int enabled);
int moba_profile_read(moba_phase_stat* stats, int max_phases);

#ifdef __cplusplus
}
#endif

#endif /* MOBA_H_ */
