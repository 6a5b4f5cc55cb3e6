// Host side of the MoBA library: argument validation, per-shape tables, the
// cached device workspace, and the order of kernel launches behind the C ABI
// declared in include/moba.h.
//
// moba_forward enqueues, on the caller's stream:
//   pool -> [bf16: V^T pack] -> gate -> route (count, column scan, bin scan,
//   scatter) -> per chunk of kv-heads: history attention, then current-block
//   attention, then the merge of the history partials (bf16: a separate
//   kernel working in place on the output; fp32: fused into the current-block
//   kernel).
// Only the attention steps depend on the chunk; their workspace (the
// partials: bf16 on the bf16 path, fp32 on the fp32 path) is what the
// workspace cap limits.
#include "moba.h"
#include "bwd_internal.h"
#include "decode_internal.h"
#include "moba_internal.h"

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

using namespace moba;

namespace {

constexpr size_t kAlign = 256;
constexpr size_t kDefaultWorkspaceLimit = size_t(64) << 30;
constexpr int kSpinLimit = 1 << 20;  // polls of a dK/dV hand-over flag before a wave gives up

// ------------------------------------------------------------- profiling
struct PhaseRec {
  const char* name;
  hipEvent_t a, b;
};
bool g_prof = false;
std::vector<PhaseRec> g_recs;
std::mutex g_prof_mu;

struct Phase {
  hipStream_t st;
  PhaseRec rec{};
  bool on = false;
  Phase(const char* name, hipStream_t s) : st(s) {
    if (!g_prof || !name) return;
    rec.name = name;
    if (hipEventCreate(&rec.a) != hipSuccess) return;
    if (hipEventCreate(&rec.b) != hipSuccess) { (void)hipEventDestroy(rec.a); return; }
    (void)hipEventRecord(rec.a, st);
    on = true;
  }
  ~Phase() {
    if (!on) return;
    (void)hipEventRecord(rec.b, st);
    std::lock_guard<std::mutex> lk(g_prof_mu);
    g_recs.push_back(rec);
  }
};

bool env_flag(const char* name) {
  const char* e = std::getenv(name);
  return e && e[0] && e[0] != '0';
}

// Read at every launch, so a process can switch it on and off.
bool debug_sync() { return env_flag("MOBA_DEBUG_SYNC"); }

#define MOBA_LAUNCH(expr)                                         \
  do {                                                            \
    hipError_t e_ = (expr);                                       \
    if (e_ != hipSuccess) return MOBA_ERR_HIP;                    \
    if (debug_sync() && hipStreamSynchronize(stream) != hipSuccess) \
      return MOBA_ERR_HIP;                                        \
  } while (0)

size_t workspace_limit() {
  const char* e = std::getenv("MOBA_WORKSPACE_LIMIT_BYTES");
  if (!e || !e[0]) return kDefaultWorkspaceLimit;
  char* end = nullptr;
  unsigned long long v = std::strtoull(e, &end, 10);
  return (end && *end == 0) ? (size_t)v : kDefaultWorkspaceLimit;
}

// ------------------------------------------------------------- validation
struct View {
  void* data;
  int64_t st, sh;  // token and head strides, elements
  int64_t H;
};

// Number of elements a descriptor spans (0 if any dimension is empty).
int64_t numel(const moba_tensor* t) {
  int64_t n = 1;
  for (int d = 0; d < t->ndim && d < 4; d++) n *= std::max<int64_t>(t->shape[d], 0);
  return n;
}

// A data pointer may be NULL only for an empty tensor.
bool missing(const moba_tensor* t) { return !t || (!t->data && (t->ndim < 1 || t->ndim > 4 || numel(t) > 0)); }

moba_status check_3d(const moba_tensor* t, int dtype, View* v) {
  if (missing(t)) return MOBA_ERR_NULL;
  if (t->dtype != dtype) return MOBA_ERR_DTYPE;
  if (t->ndim != 3) return MOBA_ERR_SHAPE;
  if (t->shape[0] < 0 || t->shape[1] < 1) return MOBA_ERR_SHAPE;
  if (t->shape[2] != kHeadDim) return MOBA_ERR_UNSUPPORTED;
  if (t->stride[2] != 1 || t->stride[0] < 0 || t->stride[1] < 0) return MOBA_ERR_LAYOUT;
  // 16-byte vector accesses: base and both strides must keep rows 16-byte aligned
  const int64_t per16 = dtype == MOBA_BF16 ? 8 : 4;
  if ((reinterpret_cast<uintptr_t>(t->data) & 15) != 0 || t->stride[0] % per16 != 0 ||
      t->stride[1] % per16 != 0)
    return MOBA_ERR_LAYOUT;
  v->data = t->data;
  v->st = t->stride[0];
  v->sh = t->stride[1];
  v->H = t->shape[1];
  return MOBA_OK;
}

moba_status check_contig(const moba_tensor* t, int dtype, int ndim, const int64_t* shape) {
  if (missing(t)) return MOBA_ERR_NULL;
  if (t->dtype != dtype) return MOBA_ERR_DTYPE;
  if (t->ndim != ndim) return MOBA_ERR_SHAPE;
  for (int d = 0; d < ndim; d++)
    if (t->shape[d] != shape[d]) return MOBA_ERR_SHAPE;
  if (numel(t) == 0) return MOBA_OK;  // strides of an empty tensor are irrelevant
  int64_t expect = 1;
  for (int d = ndim - 1; d >= 0; d--) {
    if (t->shape[d] > 1 && t->stride[d] != expect) return MOBA_ERR_LAYOUT;
    expect *= shape[d];
  }
  return MOBA_OK;
}

// Descriptor-level checks of cu_seqlens (no data access).
moba_status check_cu_desc(const moba_tensor* cu) {
  if (!cu || !cu->data) return MOBA_ERR_NULL;
  if (cu->dtype != MOBA_I32) return MOBA_ERR_DTYPE;
  if (cu->ndim != 1 || cu->shape[0] < 1) return MOBA_ERR_SHAPE;
  if (cu->shape[0] > 1 && cu->stride[0] != 1) return MOBA_ERR_LAYOUT;
  return MOBA_OK;
}

bool on_device(const void* ptr) {
  hipPointerAttribute_t attr;
  if (hipPointerGetAttributes(&attr, ptr) != hipSuccess) {
    (void)hipGetLastError();  // plain host memory
    return false;
  }
  return attr.type == hipMemoryTypeDevice || attr.type == hipMemoryTypeManaged;
}

// Pinned staging buffer for cu_seqlens that live on the device.
std::mutex g_cu_mu;
int32_t* g_cu_stage = nullptr;
int64_t g_cu_cap = 0;

// Copy cu_seqlens to the host.  Device-resident offsets are copied on the
// caller's stream, after the work that may have written them, and the
// stream is waited for (the one synchronization of such a call).
moba_status fetch_cu(const moba_tensor* cu, hipStream_t stream, std::vector<int32_t>* out) {
  const int64_t n = cu->shape[0];
  out->resize(n);
  if (on_device(cu->data)) {
    std::lock_guard<std::mutex> lk(g_cu_mu);
    if (g_cu_cap < n) {
      if (g_cu_stage) (void)hipHostFree(g_cu_stage);
      g_cu_stage = nullptr;
      g_cu_cap = 0;
      if (hipHostMalloc(reinterpret_cast<void**>(&g_cu_stage), n * sizeof(int32_t),
                        hipHostMallocDefault) != hipSuccess) {
        (void)hipGetLastError();
        g_cu_stage = nullptr;
        return MOBA_ERR_NO_MEMORY;
      }
      g_cu_cap = n;
    }
    if (hipMemcpyAsync(g_cu_stage, cu->data, n * sizeof(int32_t), hipMemcpyDeviceToHost,
                       stream) != hipSuccess ||
        hipStreamSynchronize(stream) != hipSuccess)
      return MOBA_ERR_HIP;
    std::memcpy(out->data(), g_cu_stage, n * sizeof(int32_t));
  } else {
    std::memcpy(out->data(), cu->data, n * sizeof(int32_t));
  }
  return MOBA_OK;
}

// cu[0] = 0, non-decreasing, cu[S] = T.
moba_status check_cu(const std::vector<int32_t>& c, int64_t T) {
  const int64_t n = (int64_t)c.size();
  if (c[0] != 0) return MOBA_ERR_SEQLENS;
  for (int64_t s = 0; s + 1 < n; s++)
    if (c[s + 1] < c[s]) return MOBA_ERR_SEQLENS;
  if (c[n - 1] != T) return MOBA_ERR_SEQLENS;
  return MOBA_OK;
}

moba_status read_cu(const moba_tensor* cu, int64_t T, hipStream_t stream,
                    std::vector<int32_t>* out) {
  moba_status st = fetch_cu(cu, stream, out);
  return st != MOBA_OK ? st : check_cu(*out, T);
}

// ------------------------------------------------------------- planning
enum TileMode { kTilesNone = 0, kTilesCur = 1, kTilesDense = 2 };

struct Plan {
  Problem p{};
  std::vector<SeqInfo> seqs;
  std::vector<CausalTile> tiles;
  std::vector<KeyTile> ktiles;  // key tiles of the dK/dV kernel (kTilesCur plans)
  int64_t hist_per_head = 0;  // history selections of one query head, summed over tokens
};

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// B = 0 means "one block per sequence" (dense attention).
void build_plan(const std::vector<int32_t>& cu, int Hq, int Hkv, int B, int topk, TileMode mode,
                int tile_rows, Plan* pl) {
  Problem& p = pl->p;
  const int S = (int)cu.size() - 1;
  p.T = cu[S];
  p.Hq = Hq;
  p.Hkv = Hkv;
  p.G = Hq / Hkv;
  p.S = S;
  p.B = B;
  p.topk = topk;
  p.tile_rows = tile_rows;
  p.gate_tw = std::max(1, 256 / p.G);
  p.route_rt = std::max(1, kRouteRows / p.G);
  p.sel_st = Hq;  // the callers' [T, Hq, topk]
  p.sel_sg = p.G;
  pl->seqs.assign(S, SeqInfo{});
  int64_t blk = 0, vt = 0, gate = 0, rc = 0, hw = 0, hist = 0;
  int nbmax = 0;
  const int64_t kh = topk - 1;
  for (int s = 0; s < S; s++) {
    SeqInfo& q = pl->seqs[s];
    const int64_t L = (int64_t)cu[s + 1] - cu[s];
    const int64_t Bs = B > 0 ? B : std::max<int64_t>(L, 1);
    const int64_t nb = ceil_div(L, Bs);
    q.tok_start = cu[s];
    q.len = (int32_t)L;
    q.blk_off = (int32_t)blk;
    q.nblk = (int32_t)nb;
    q.vt_tile_off = (int32_t)vt;
    q.gate_off = (int32_t)gate;
    q.rc_off = (int32_t)rc;
    q.hist_off = hw;
    blk += nb;
    vt += ceil_div(L, kKeyTile);
    gate += ceil_div(L, p.gate_tw);
    rc += ceil_div(L, p.route_rt);
    hw += ceil_div(L, p.route_rt) * nb;
    nbmax = std::max<int>(nbmax, (int)nb);
    if (B > 0)
      for (int64_t c = 0; c < nb; c++) {
        const int64_t m = std::min<int64_t>(L, (c + 1) * B) - c * B;
        hist += m * std::min<int64_t>(kh, c);
      }
  }
  p.nblk_total = (int)blk;
  p.nblk_max = nbmax;
  p.vt_tiles = vt;
  p.gate_groups = gate;
  p.route_chunks = rc;
  p.hist_words = hw;
  pl->hist_per_head = hist;
  p.hist_entries = hist * Hq;

  pl->tiles.clear();
  pl->ktiles.clear();
  if (mode == kTilesNone) return;
  const int tt = std::max(1, tile_rows / p.G);  // tokens per causal tile
  if (mode == kTilesCur) {
    // Tiles of one key block read the same K/V.  Work-groups go round-robin
    // to the 8 XCDs (each with its own L2), so each block's tiles are put on
    // one XCD, longest first, with blocks spread greedily over the XCDs by
    // key work; tile x of the list runs on XCD x % 8 (the list is padded
    // with empty tiles to a multiple of 8).
    struct Group { int64_t work; std::vector<CausalTile> tiles; };
    std::vector<Group> groups;
    for (int s = 0; s < S; s++) {
      const int64_t L = (int64_t)cu[s + 1] - cu[s];
      for (int64_t b0 = 0; b0 < L; b0 += B) {
        const int64_t b1 = std::min(L, b0 + B);
        Group gr{0, {}};
        for (int64_t t0 = b0; t0 < b1; t0 += tt) {
          const int64_t t1 = std::min(b1, t0 + tt);
          gr.tiles.push_back(CausalTile{s, (int32_t)(cu[s] + t0), (int32_t)(cu[s] + t1),
                                        (int32_t)(cu[s] + b0)});
          gr.work += t1 - b0;
        }
        std::reverse(gr.tiles.begin(), gr.tiles.end());
        groups.push_back(std::move(gr));
      }
    }
    std::stable_sort(groups.begin(), groups.end(),
                     [](const Group& x, const Group& y) { return x.work > y.work; });
    constexpr int kXcd = 8;
    std::vector<std::vector<CausalTile>> lists(kXcd);
    int64_t load[kXcd] = {0};
    for (const Group& gr : groups) {
      const int x = (int)(std::min_element(load, load + kXcd) - load);
      lists[x].insert(lists[x].end(), gr.tiles.begin(), gr.tiles.end());
      load[x] += gr.work;
    }
    size_t n = 0;
    for (const auto& l : lists) n = std::max(n, l.size());
    for (size_t k = 0; k < n; k++)
      for (int x = 0; x < kXcd; x++)
        pl->tiles.push_back(k < lists[x].size() ? lists[x][k] : CausalTile{0, 0, 0, 0});
    // dK/dV key tiles: local block 0 of every sequence first (early blocks
    // collect the longest routed row lists), then block 1, ...
    for (int j = 0; j < nbmax; j++)
      for (int s = 0; s < S; s++) {
        const int64_t L = (int64_t)cu[s + 1] - cu[s];
        const int64_t b0 = (int64_t)j * B;
        if (b0 >= L) continue;
        const int64_t b1 = std::min(L, b0 + B);
        for (int64_t k0 = b0; k0 < b1; k0 += kKeysPerDkdv)
          pl->ktiles.push_back(KeyTile{pl->seqs[s].blk_off + j, (int32_t)(cu[s] + k0),
                                       (int32_t)(cu[s] + std::min(b1, k0 + kKeysPerDkdv)),
                                       (int32_t)(cu[s] + b1)});
      }
    return;
  }
  for (int s = 0; s < S; s++) {
    const int64_t L = (int64_t)cu[s + 1] - cu[s];
    const int64_t Bs = std::max<int64_t>(L, 1);
    for (int64_t b0 = 0; b0 < L; b0 += Bs) {
      const int64_t b1 = std::min(L, b0 + Bs);
      for (int64_t t0 = b0; t0 < b1; t0 += tt)
        pl->tiles.push_back(CausalTile{s, (int32_t)(cu[s] + t0),
                                       (int32_t)(cu[s] + std::min(b1, t0 + tt)),
                                       (int32_t)(cu[s] + b0)});
    }
  }
  // longest key range first, so the long tiles start early
  std::stable_sort(pl->tiles.begin(), pl->tiles.end(), [](const CausalTile& x, const CausalTile& y) {
    return (x.t1 - x.kbeg) > (y.t1 - y.kbeg);
  });
}

// ------------------------------------------------------------- device cache
// A plan with its tables on the device.  The tables are built in pinned host
// memory and copied on the caller's stream, so a new plan needs no device
// synchronization: the copy runs after every earlier call's kernels (stream
// order, and calls on different streams never overlap), and `uploaded` tells
// when the staging buffer may be written again.
struct PlanSlot {
  std::vector<int64_t> key;  // empty: unused
  Plan plan;
  void* tab = nullptr;       // device tables
  size_t tab_bytes = 0;
  void* stage = nullptr;     // pinned host copy of the tables
  size_t stage_bytes = 0;
  hipEvent_t uploaded = nullptr;
  bool pending = false;      // `uploaded` recorded after the last copy
  uint64_t last_use = 0;
};
constexpr int kPlanSlots = 4;  // e.g. forward/backward, decode, and the step-level calls

struct DevCache {
  void* ws = nullptr;
  size_t ws_bytes = 0;
  PlanSlot slots[kPlanSlots];
  uint64_t clock = 0;
  uint32_t* wait_timeouts = nullptr;  // device counter of dK/dV hand-over give-ups
};
std::mutex g_mu;
std::map<int, DevCache> g_dev;

DevCache* cache_for_current_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return nullptr;
  return &g_dev[dev];
}

moba_status ensure_workspace(DevCache* dc, size_t bytes) {
  if (bytes <= dc->ws_bytes) return MOBA_OK;
  if (dc->ws) {
    if (hipDeviceSynchronize() != hipSuccess) return MOBA_ERR_HIP;
    (void)hipFree(dc->ws);
    dc->ws = nullptr;
    dc->ws_bytes = 0;
  }
  const size_t sz = (bytes + (size_t(1) << 20) - 1) & ~((size_t(1) << 20) - 1);
  if (hipMalloc(&dc->ws, sz) != hipSuccess) {
    (void)hipGetLastError();
    dc->ws = nullptr;
    return MOBA_ERR_NO_MEMORY;
  }
  dc->ws_bytes = sz;
  return MOBA_OK;
}

// ------------------------------------------------------------- no-alloc scratch
// moba_decode_noalloc's buffers: a static device array per GPU (held from
// module load until the process ends).  Host code never passes the array's
// name to a kernel: its device address is looked up once per device.
constexpr size_t kNoAllocScratchBytes = MOBA_DECODE_NOALLOC_MAX_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

std::mutex g_na_mu;
std::map<int, char*> g_na_ptr;  // device -> address of `scratch` on it

moba_status noalloc_scratch(char** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MOBA_ERR_HIP;
  std::lock_guard<std::mutex> lk(g_na_mu);
  auto it = g_na_ptr.find(dev);
  if (it == g_na_ptr.end()) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return MOBA_ERR_HIP;
    }
    it = g_na_ptr.emplace(dev, static_cast<char*>(p)).first;
  }
  *out = it->second;
  return MOBA_OK;
}

// Per-sequence tables passed to the device by value (kernel arguments).
constexpr int kSeqsPerCopy = 32;
struct SeqBatch {
  SeqInfo s[kSeqsPerCopy];
  int32_t n;
};

__global__ void seq_table_kernel(SeqBatch b, SeqInfo* dst) {
  const int i = threadIdx.x;
  if (i < b.n) dst[i] = b.s[i];
}

hipError_t launch_seq_table(const SeqBatch& b, SeqInfo* dst, hipStream_t st) {
  seq_table_kernel<<<1, kSeqsPerCopy, 0, st>>>(b, dst);
  return hipGetLastError();
}

// The device's give-up counter of the dK/dV hand-over wait, zeroed when made.
moba_status ensure_wait_counter(DevCache* dc) {
  if (dc->wait_timeouts) return MOBA_OK;
  void* p = nullptr;
  if (hipMalloc(&p, kAlign) != hipSuccess) {
    (void)hipGetLastError();
    return MOBA_ERR_NO_MEMORY;
  }
  if (hipMemset(p, 0, kAlign) != hipSuccess) {
    (void)hipFree(p);
    return MOBA_ERR_HIP;
  }
  dc->wait_timeouts = static_cast<uint32_t*>(p);
  return MOBA_OK;
}

// Reads and clears the give-up counter (synchronous).
moba_status take_wait_counter(DevCache* dc, uint64_t* count) {
  *count = 0;
  if (!dc->wait_timeouts) return MOBA_OK;
  uint32_t v = 0;
  if (hipDeviceSynchronize() != hipSuccess ||
      hipMemcpy(&v, dc->wait_timeouts, sizeof(v), hipMemcpyDeviceToHost) != hipSuccess ||
      hipMemset(dc->wait_timeouts, 0, sizeof(v)) != hipSuccess)
    return MOBA_ERR_HIP;
  *count = v;
  return MOBA_OK;
}

// Plan for (cu, heads, B, topk, mode), with its tables resident on the device.
// Kept in a small least-recently-used set of slots, so calls that alternate
// between a few shapes rebuild nothing.  A rebuild copies the tables on
// `stream` without synchronizing the device (only growing a slot's buffers
// does).
moba_status get_plan(DevCache* dc, hipStream_t stream, const std::vector<int32_t>& cu, int Hq,
                     int Hkv, int B, int topk, TileMode mode, int tile_rows, const Plan** out,
                     const SeqInfo** d_seqs, const CausalTile** d_tiles,
                     const KeyTile** d_ktiles = nullptr) {
  std::vector<int64_t> key = {Hq, Hkv, B, topk, mode, tile_rows, (int64_t)cu.size()};
  key.insert(key.end(), cu.begin(), cu.end());
  PlanSlot* sl = nullptr;
  for (PlanSlot& x : dc->slots)
    if (!x.key.empty() && x.key == key) sl = &x;
  if (!sl) {
    sl = &dc->slots[0];
    for (PlanSlot& x : dc->slots)
      if (x.key.empty() || x.last_use < sl->last_use) sl = &x;
    // the slot's previous copy must have read its staging buffer
    if (sl->pending && hipEventSynchronize(sl->uploaded) != hipSuccess) return MOBA_ERR_HIP;
    sl->pending = false;
    sl->key.clear();
    Plan pl;
    build_plan(cu, Hq, Hkv, B, topk, mode, tile_rows, &pl);
    const size_t sb = pl.seqs.size() * sizeof(SeqInfo);
    const size_t tb = pl.tiles.size() * sizeof(CausalTile);
    const size_t toff = ((sb + kAlign - 1) / kAlign) * kAlign;
    const size_t koff = toff + ((tb + kAlign - 1) / kAlign) * kAlign;
    const size_t need = koff + pl.ktiles.size() * sizeof(KeyTile);
    // buffers grow to a power of two (at least 64 KiB), so a growing cache
    // rarely reallocates
    size_t cap = size_t(1) << 16;
    while (cap < need) cap <<= 1;
    if (need > sl->tab_bytes || !sl->tab) {
      // kernels of earlier calls may still read the old tables
      if (hipDeviceSynchronize() != hipSuccess) return MOBA_ERR_HIP;
      if (sl->tab) (void)hipFree(sl->tab);
      sl->tab = nullptr;
      sl->tab_bytes = 0;
      if (hipMalloc(&sl->tab, cap) != hipSuccess) {
        (void)hipGetLastError();
        sl->tab = nullptr;
        return MOBA_ERR_NO_MEMORY;
      }
      sl->tab_bytes = cap;
    }
    if (need > sl->stage_bytes || !sl->stage) {
      if (sl->stage) (void)hipHostFree(sl->stage);
      sl->stage = nullptr;
      sl->stage_bytes = 0;
      if (hipHostMalloc(&sl->stage, cap, hipHostMallocDefault) != hipSuccess) {
        (void)hipGetLastError();
        sl->stage = nullptr;
        return MOBA_ERR_NO_MEMORY;
      }
      sl->stage_bytes = cap;
    }
    if (!sl->uploaded && hipEventCreateWithFlags(&sl->uploaded, hipEventDisableTiming) != hipSuccess) {
      sl->uploaded = nullptr;
      return MOBA_ERR_HIP;
    }
    char* st = static_cast<char*>(sl->stage);
    if (sb) std::memcpy(st, pl.seqs.data(), sb);
    if (tb) std::memcpy(st + toff, pl.tiles.data(), tb);
    if (!pl.ktiles.empty()) std::memcpy(st + koff, pl.ktiles.data(), pl.ktiles.size() * sizeof(KeyTile));
    if (need && (hipMemcpyAsync(sl->tab, sl->stage, need, hipMemcpyHostToDevice, stream) != hipSuccess ||
                 hipEventRecord(sl->uploaded, stream) != hipSuccess))
      return MOBA_ERR_HIP;
    sl->pending = need != 0;
    sl->plan = std::move(pl);
    sl->key = std::move(key);
  }
  sl->last_use = ++dc->clock;
  const size_t sb = sl->plan.seqs.size() * sizeof(SeqInfo);
  const size_t tb = sl->plan.tiles.size() * sizeof(CausalTile);
  const size_t toff = ((sb + kAlign - 1) / kAlign) * kAlign;
  *out = &sl->plan;
  *d_seqs = static_cast<const SeqInfo*>(sl->tab);
  *d_tiles = reinterpret_cast<const CausalTile*>(static_cast<char*>(sl->tab) + toff);
  if (d_ktiles)
    *d_ktiles = reinterpret_cast<const KeyTile*>(static_cast<char*>(sl->tab) + toff +
                                                 ((tb + kAlign - 1) / kAlign) * kAlign);
  return MOBA_OK;
}

// Bump allocator over the workspace; the first pass (base == nullptr) sizes it.
struct Bump {
  char* base;
  size_t off = 0;
  explicit Bump(void* b) : base(static_cast<char*>(b)) {}
  template <typename T>
  T* take(int64_t n) {
    off = (off + kAlign - 1) / kAlign * kAlign;
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += (size_t)std::max<int64_t>(n, 0) * sizeof(T);
    return p;
  }
};

struct Inputs {
  View q, k, v;
  bool bf16;
  int64_t T;
  int Hq, Hkv;
  std::vector<int32_t> cu;
};

// Checks shared by moba_forward and moba_dense_forward.
moba_status check_inputs(const moba_tensor* q, const moba_tensor* k, const moba_tensor* v,
                         const moba_tensor* cu, const moba_tensor* out, const moba_tensor* lse,
                         Inputs* in, View* vo) {
  if (missing(q) || missing(k) || missing(v) || missing(out) || missing(lse) || !cu || !cu->data)
    return MOBA_ERR_NULL;
  if (q->dtype != MOBA_BF16 && q->dtype != MOBA_F32) return MOBA_ERR_DTYPE;
  moba_status st;
  if ((st = check_3d(q, q->dtype, &in->q)) != MOBA_OK) return st;
  if ((st = check_3d(k, q->dtype, &in->k)) != MOBA_OK) return st;
  if ((st = check_3d(v, q->dtype, &in->v)) != MOBA_OK) return st;
  if ((st = check_3d(out, q->dtype, vo)) != MOBA_OK) return st;
  in->T = q->shape[0];
  in->Hq = (int)q->shape[1];
  in->Hkv = (int)k->shape[1];
  if (k->shape[0] != in->T || v->shape[0] != in->T || out->shape[0] != in->T) return MOBA_ERR_SHAPE;
  if (v->shape[1] != in->Hkv || out->shape[1] != in->Hq) return MOBA_ERR_SHAPE;
  if (in->Hq % in->Hkv != 0) return MOBA_ERR_SHAPE;
  if (in->Hq / in->Hkv > kMaxGroup) return MOBA_ERR_UNSUPPORTED;
  const int64_t lshape[2] = {in->Hq, in->T};
  if ((st = check_contig(lse, MOBA_F32, 2, lshape)) != MOBA_OK) return st;
  if ((st = check_cu_desc(cu)) != MOBA_OK) return st;
  if (in->T >= (int64_t(1) << 31) - kTileRowsMfma) return MOBA_ERR_UNSUPPORTED;
  in->bf16 = q->dtype == MOBA_BF16;
  return MOBA_OK;
}

AttnArgs make_args(const Inputs& in, const View& vo, float* lse) {
  AttnArgs a{};
  a.q = in.q.data; a.q_st = in.q.st; a.q_sh = in.q.sh;
  a.k = in.k.data; a.k_st = in.k.st; a.k_sh = in.k.sh;
  a.v = in.v.data; a.v_st = in.v.st; a.v_sh = in.v.sh;
  a.out = vo.data; a.o_st = vo.st; a.o_sh = vo.sh;
  a.lse = lse;
  a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)kHeadDim));
  return a;
}

moba_status dense_forward_impl(const Inputs& in, const View& vo, moba_tensor* lse,
                               hipStream_t stream);

// The forward's workspace: a fixed part (block keys, packed V^T, selection,
// routing lists) and a part per chunk of `nch` kv-heads (the history
// partials and their lse).
struct FwdBufs {
  float* kbar;
  __hip_bfloat16* kterm;  // bf16 path: the three exact bf16 planes of kbar
  __hip_bfloat16* vt;
  int32_t* sel;
  RouteBuffers rb;
  void* o_part;
  float* lse_part;
};

void forward_layout(const Problem& p, bool bf16, int kk, int nch, Bump* bp, FwdBufs* b) {
  const int64_t kh = kk - 1;
  const int64_t nbins = (int64_t)p.Hkv * p.nblk_total;
  b->kbar = bp->take<float>((int64_t)p.nblk_total * p.Hkv * kHeadDim);
  b->kterm = bf16 ? bp->take<__hip_bfloat16>((int64_t)3 * p.nblk_total * p.Hkv * kHeadDim) : nullptr;
  b->vt = bf16 ? bp->take<__hip_bfloat16>((int64_t)p.Hkv * p.vt_tiles * kKeyTile * kHeadDim) : nullptr;
  b->sel = bp->take<int32_t>(p.T * p.Hq * kk);
  b->rb.hist = bp->take<int32_t>((int64_t)p.Hkv * p.hist_words);
  b->rb.bin_count = bp->take<int32_t>(nbins);
  b->rb.bin_start = bp->take<int64_t>(nbins + 1);
  b->rb.bin_tile_start = bp->take<int32_t>(nbins + 1);
  b->rb.entries = bp->take<uint32_t>(p.hist_entries);
  b->rb.tile_bin = bp->take<int32_t>(route_tiles_bound(p.hist_entries, nbins, p.tile_rows));
  const int64_t rows = (int64_t)nch * p.T * p.G;
  b->o_part = bf16 ? (void*)bp->take<__hip_bfloat16>(rows * kh * kHeadDim)
                   : (void*)bp->take<float>(rows * kh * kHeadDim);
  b->lse_part = bp->take<float>(rows * kh);
}

// Number of blocks and of history selections (route entries) of a batch:
// sum over sequences of ceil(L / B), and Hq times the sum over tokens of
// min(topk - 1, c), c the token's block (Eq. 5 keeps min(k - 1, c) past
// blocks besides the current one).
void batch_sizes(const std::vector<int32_t>& cu, int B, int topk, int Hq, int64_t* nblk,
                 int64_t* entries) {
  int64_t nb = 0, e = 0;
  for (size_t s = 0; s + 1 < cu.size(); s++) {
    const int64_t L = (int64_t)cu[s + 1] - cu[s];
    const int64_t n = ceil_div(L, B);
    nb += n;
    for (int64_t c = 0; c < n; c++)
      e += (std::min<int64_t>(L, (c + 1) * B) - c * B) * std::min<int64_t>(topk - 1, c);
  }
  *nblk = nb;
  *entries = e * Hq;
}

}  // namespace

// ======================================================================= ABI
extern "C" {

moba_status moba_forward(const moba_tensor* q, const moba_tensor* k, const moba_tensor* v,
                         const moba_tensor* cu_seqlens, int32_t block_size, int32_t topk,
                         moba_tensor* out, moba_tensor* lse, hipStream_t stream) {
  Inputs in;
  View vo;
  moba_status st = check_inputs(q, k, v, cu_seqlens, out, lse, &in, &vo);
  if (st != MOBA_OK) return st;
  if (block_size < 1) return MOBA_ERR_BLOCK_SIZE;
  if (topk < 1) return MOBA_ERR_TOPK;
  if ((st = read_cu(cu_seqlens, in.T, stream, &in.cu)) != MOBA_OK) return st;
  if (in.T == 0) return MOBA_OK;

  // blocks per sequence and the effective top-k (more than #blocks changes nothing)
  int64_t nbmax = 0;
  for (size_t s = 0; s + 1 < in.cu.size(); s++)
    nbmax = std::max<int64_t>(nbmax, ceil_div((int64_t)in.cu[s + 1] - in.cu[s], block_size));
  // top-k covering every block of every sequence selects each row's whole
  // causal prefix (Eq. 5 keeps all min(k, c + 1) blocks): full attention
  if (topk >= nbmax) return dense_forward_impl(in, vo, lse, stream);
  if (nbmax > kMaxBlocksPerSeq) return MOBA_ERR_UNSUPPORTED;
  const int kk = (int)std::min<int64_t>(topk, nbmax);
  if (kk - 1 > 63 && kk - 1 < nbmax - 1) return MOBA_ERR_UNSUPPORTED;
  if ((uint64_t)in.T * in.Hq * (uint64_t)std::max(kk - 1, 1) >= (uint64_t(1) << 32))
    return MOBA_ERR_UNSUPPORTED;

  std::lock_guard<std::mutex> lk(g_mu);
  DevCache* dc = cache_for_current_device();
  if (!dc) return MOBA_ERR_HIP;
  const Plan* pl;
  const SeqInfo* d_seqs;
  const CausalTile* d_tiles;
  if ((st = get_plan(dc, stream, in.cu, in.Hq, in.Hkv, block_size, kk, kTilesCur,
                     in.bf16 ? kTileRowsMfma : kTileRowsF32, &pl, &d_seqs, &d_tiles)) !=
      MOBA_OK)
    return st;
  Problem p = pl->p;  // the selection is private here: kv-head-major
  p.sel_st = p.G;
  p.sel_sg = p.T * p.G;
  const int64_t kh = kk - 1;

  // workspace: fixed part, then per-kv-head chunk part
  const size_t limit = workspace_limit();
  int nch = 0;
  size_t need = 0;
  for (int n = p.Hkv; n >= 1; n--) {
    Bump bp(nullptr);
    FwdBufs b{};
    forward_layout(p, in.bf16, kk, n, &bp, &b);
    if (bp.off + kAlign <= limit) { nch = n; need = bp.off + kAlign; break; }
  }
  if (nch == 0) return MOBA_ERR_NO_MEMORY;
  // as many chunks as the cap requires, of equal size (the last may be smaller)
  nch = (int)ceil_div(p.Hkv, ceil_div(p.Hkv, nch));
  if ((st = ensure_workspace(dc, need)) != MOBA_OK) return st;

  Bump bp(dc->ws);
  AttnArgs a = make_args(in, vo, static_cast<float*>(lse->data));
  FwdBufs fb{};
  forward_layout(p, in.bf16, kk, nch, &bp, &fb);
  RouteBuffers rb = fb.rb;
  float* kbar = fb.kbar;
  __hip_bfloat16* vt = fb.vt;
  int32_t* sel = fb.sel;
  a.o_part = fb.o_part;
  a.lse_part = fb.lse_part;
  a.vt = vt;
  a.seqs = d_seqs;
  a.bin_tile_start = rb.bin_tile_start;
  a.tile_bin = rb.tile_bin;
  a.bin_start = rb.bin_start;
  a.bin_count = rb.bin_count;
  a.entries = rb.entries;
  a.tiles = d_tiles;
  a.ntiles = (int64_t)pl->tiles.size();

  { Phase ph("pool", stream);
    MOBA_LAUNCH(launch_pool(in.k.data, in.bf16, in.k.st, in.k.sh, d_seqs, p, kbar, fb.kterm,
                            stream)); }
  if (in.bf16) {
    Phase ph("vt_pack", stream);
    MOBA_LAUNCH(launch_vt_pack(static_cast<const __hip_bfloat16*>(in.v.data), in.v.st, in.v.sh,
                               d_seqs, p, vt, stream));
  }
  { Phase ph("gate", stream);
    MOBA_LAUNCH(launch_gate(in.q.data, in.bf16, in.q.st, in.q.sh, kbar, fb.kterm, d_seqs, p, sel,
                            nullptr, 0,
                            stream)); }
  if (kh > 0 && p.hist_entries > 0) {
    Phase ph("route", stream);
    MOBA_LAUNCH(launch_route(sel, d_seqs, p, rb, stream));
  }
  for (int g0 = 0; g0 < p.Hkv; g0 += nch) {
    a.g0 = g0;
    a.g1 = std::min(p.Hkv, g0 + nch);
    const int64_t e_chunk = pl->hist_per_head * p.G * (a.g1 - a.g0);
    if (kh > 0 && e_chunk > 0) {
      const int64_t grid = ceil_div(e_chunk, p.tile_rows) + (int64_t)(a.g1 - a.g0) * p.nblk_total;
      Phase ph("attn_hist", stream);
      MOBA_LAUNCH(in.bf16 ? launch_attn_hist_bf16(a, p, grid, stream)
                          : launch_attn_hist_f32(a, p, grid, stream));
    }
    if (in.bf16) {
      { Phase ph("attn_cur", stream);
        MOBA_LAUNCH(launch_attn_causal_bf16(false, a, p, stream)); }
      if (kh > 0) {
        Phase ph("merge", stream);
        MOBA_LAUNCH(launch_merge_bf16(a, p, stream));
      }
    } else {
      Phase ph("attn_cur_merge", stream);
      MOBA_LAUNCH(launch_attn_causal_f32(false, a, p, stream));
    }
  }
  return MOBA_OK;
}

}  // extern "C"

namespace {

// The backward of moba_forward; with `dense`, of moba_dense_forward (each
// sequence one block, top-1: the causal current block is the whole prefix).
moba_status backward_impl(const moba_tensor* q, const moba_tensor* k, const moba_tensor* v,
                          const moba_tensor* cu_seqlens, int32_t block_size, int32_t topk,
                          const moba_tensor* out, const moba_tensor* lse, const moba_tensor* dout,
                          moba_tensor* dq, moba_tensor* dk, moba_tensor* dv, hipStream_t stream,
                          bool dense) {
  Inputs in;
  View vo, vdo, vdq, vdk, vdv;
  moba_status st = check_inputs(q, k, v, cu_seqlens, out, lse, &in, &vo);
  if (st != MOBA_OK) return st;
  if (!in.bf16) return MOBA_ERR_DTYPE;
  if (missing(dout) || missing(dq) || missing(dk) || missing(dv)) return MOBA_ERR_NULL;
  if ((st = check_3d(dout, MOBA_BF16, &vdo)) != MOBA_OK) return st;
  if ((st = check_3d(dq, MOBA_BF16, &vdq)) != MOBA_OK) return st;
  if ((st = check_3d(dk, MOBA_BF16, &vdk)) != MOBA_OK) return st;
  if ((st = check_3d(dv, MOBA_BF16, &vdv)) != MOBA_OK) return st;
  if (dout->shape[0] != in.T || dq->shape[0] != in.T || dk->shape[0] != in.T ||
      dv->shape[0] != in.T)
    return MOBA_ERR_SHAPE;
  if (vdo.H != in.Hq || vdq.H != in.Hq || vdk.H != in.Hkv || vdv.H != in.Hkv) return MOBA_ERR_SHAPE;
  if (!dense && block_size < 1) return MOBA_ERR_BLOCK_SIZE;
  if (!dense && topk < 1) return MOBA_ERR_TOPK;
  if ((st = read_cu(cu_seqlens, in.T, stream, &in.cu)) != MOBA_OK) return st;
  if (in.T == 0) return MOBA_OK;
  if (!dense) {
    // as in the forward: top-k covering every block is full attention
    int64_t nb = 0;
    for (size_t s = 0; s + 1 < in.cu.size(); s++)
      nb = std::max<int64_t>(nb, ceil_div((int64_t)in.cu[s + 1] - in.cu[s], block_size));
    dense = topk >= nb;
  }
  if (dense) {
    int64_t lmax = 1;
    for (size_t s = 0; s + 1 < in.cu.size(); s++)
      lmax = std::max<int64_t>(lmax, (int64_t)in.cu[s + 1] - in.cu[s]);
    block_size = (int32_t)lmax;
    topk = 1;
  }

  int64_t nbmax = 0;
  for (size_t s = 0; s + 1 < in.cu.size(); s++)
    nbmax = std::max<int64_t>(nbmax, ceil_div((int64_t)in.cu[s + 1] - in.cu[s], block_size));
  if (nbmax > kMaxBlocksPerSeq) return MOBA_ERR_UNSUPPORTED;
  const int kk = (int)std::max<int64_t>(1, std::min<int64_t>(topk, nbmax));
  if (kk - 1 > 63 && kk - 1 < nbmax - 1) return MOBA_ERR_UNSUPPORTED;
  if ((uint64_t)in.T * in.Hq * (uint64_t)std::max(kk - 1, 1) >= (uint64_t(1) << 32))
    return MOBA_ERR_UNSUPPORTED;

  std::lock_guard<std::mutex> lk(g_mu);
  DevCache* dc = cache_for_current_device();
  if (!dc) return MOBA_ERR_HIP;
  const Plan* pl;
  const SeqInfo* d_seqs;
  const CausalTile* d_tiles;
  const KeyTile* d_ktiles;
  if ((st = get_plan(dc, stream, in.cu, in.Hq, in.Hkv, block_size, kk, kTilesCur, kTileRowsMfma, &pl,
                     &d_seqs, &d_tiles, &d_ktiles)) != MOBA_OK)
    return st;
  Problem p = pl->p;  // the selection is private here: kv-head-major
  p.sel_st = p.G;
  p.sel_sg = p.T * p.G;
  const int64_t kh = kk - 1;
  const int64_t TG = p.T * p.G;
  const int64_t nbins = (int64_t)p.Hkv * p.nblk_total;
  const bool routed = kh > 0 && p.hist_entries > 0;

  struct Bufs {
    float* kbar; __hip_bfloat16* kterm; __hip_bfloat16* kt; int32_t* sel; RouteBuffers rb;
    float2* ld; int4* rec;
    float* dq_part;
  };
  auto layout = [&](int nch, Bump* bp, Bufs* b) {
    b->kbar = bp->take<float>((int64_t)p.nblk_total * p.Hkv * kHeadDim);
    b->kterm = bp->take<__hip_bfloat16>((int64_t)3 * p.nblk_total * p.Hkv * kHeadDim);
    b->kt = bp->take<__hip_bfloat16>((int64_t)p.Hkv * p.vt_tiles * kKeyTile * kHeadDim);
    b->sel = bp->take<int32_t>(p.T * p.Hq * kk);
    b->rb.hist = bp->take<int32_t>((int64_t)p.Hkv * p.hist_words);
    b->rb.bin_count = bp->take<int32_t>(nbins);
    b->rb.bin_start = bp->take<int64_t>(nbins + 1);
    b->rb.bin_tile_start = bp->take<int32_t>(nbins + 1);
    b->rb.entries = bp->take<uint32_t>(p.hist_entries);
    b->rb.tile_bin = bp->take<int32_t>(route_tiles_bound(p.hist_entries, nbins, kTileRowsMfma));
    b->ld = bp->take<float2>(p.T * p.Hq);
    b->rec = bp->take<int4>(routed ? p.hist_entries : 0);
    b->dq_part = bp->take<float>(routed ? (int64_t)nch * TG * kh * kHeadDim : 0);
  };
  const size_t limit = workspace_limit();
  int nch = 0;
  size_t need = 0;
  for (int n = p.Hkv; n >= 1; n--) {
    Bump bp(nullptr);
    Bufs b{};
    layout(n, &bp, &b);
    if (bp.off + kAlign <= limit) { nch = n; need = bp.off + kAlign; break; }
  }
  if (nch == 0) return MOBA_ERR_NO_MEMORY;
  nch = (int)ceil_div(p.Hkv, ceil_div(p.Hkv, nch));
  if ((st = ensure_workspace(dc, need)) != MOBA_OK) return st;
  Bump bp(dc->ws);
  Bufs b{};
  layout(nch, &bp, &b);

  BwdArgs a{};
  a.q = in.q.data; a.q_st = in.q.st; a.q_sh = in.q.sh;
  a.k = in.k.data; a.k_st = in.k.st; a.k_sh = in.k.sh;
  a.v = in.v.data; a.v_st = in.v.st; a.v_sh = in.v.sh;
  a.o = vo.data; a.o_st = vo.st; a.o_sh = vo.sh;
  a.dout = vdo.data; a.do_st = vdo.st; a.do_sh = vdo.sh;
  a.lse = static_cast<const float*>(lse->data);
  a.dq = vdq.data; a.dq_st = vdq.st; a.dq_sh = vdq.sh;
  a.dk = vdk.data; a.dk_st = vdk.st; a.dk_sh = vdk.sh;
  a.dv = vdv.data; a.dv_st = vdv.st; a.dv_sh = vdv.sh;
  a.kt = b.kt;
  a.seqs = d_seqs;
  if (routed) {
    a.bin_tile_start = b.rb.bin_tile_start;
    a.tile_bin = b.rb.tile_bin;
    a.bin_start = b.rb.bin_start;
    a.bin_count = b.rb.bin_count;
    a.entries = b.rb.entries;
  }
  a.ld = b.ld;
  a.rec = b.rec;
  a.dq_part = b.dq_part;
  a.tiles = d_tiles;
  a.ntiles = (int64_t)pl->tiles.size();
  a.ktiles = d_ktiles;
  a.nktiles = (int64_t)pl->ktiles.size();
  a.scale = (float)(1.0 / std::sqrt((double)kHeadDim));
  a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)kHeadDim));
  if ((st = ensure_wait_counter(dc)) != MOBA_OK) return st;
  a.wait_timeouts = dc->wait_timeouts;
  a.spin_limit = kSpinLimit;
  a.wait_bias = 0;
  if (env_flag("MOBA_FORCE_WAIT_TIMEOUT")) {
    // testing aid: every hand-over wait gives up after a few polls (the
    // kernel still runs to its end; the gradients are then wrong)
    a.spin_limit = 64;
    a.wait_bias = 1 << 30;
  }

  // the forward's selection and routing, recomputed
  { Phase ph("pool", stream);
    MOBA_LAUNCH(launch_pool(in.k.data, true, in.k.st, in.k.sh, d_seqs, p, b.kbar, b.kterm,
                            stream)); }
  { Phase ph("kt_pack", stream);
    MOBA_LAUNCH(launch_vt_pack(static_cast<const __hip_bfloat16*>(in.k.data), in.k.st, in.k.sh,
                               d_seqs, p, b.kt, stream)); }
  { Phase ph("gate", stream);
    MOBA_LAUNCH(launch_gate(in.q.data, true, in.q.st, in.q.sh, b.kbar, b.kterm, d_seqs, p, b.sel,
                            nullptr, 0,
                            stream)); }
  if (routed) {
    Phase ph("route", stream);
    MOBA_LAUNCH(launch_route(b.sel, d_seqs, p, b.rb, stream));
  }
  { Phase ph("bwd_delta", stream);
    MOBA_LAUNCH(launch_bwd_delta(a, p, stream)); }
  if (routed) {
    Phase ph("bwd_rec", stream);
    MOBA_LAUNCH(launch_bwd_rec(a, p, stream));
  }
  { Phase ph("bwd_dkdv", stream);
    MOBA_LAUNCH(launch_bwd_dkdv(a, p, stream)); }
  if (debug_sync()) {
    // the launch above has completed: report a hand-over wait that gave up
    uint64_t n = 0;
    if ((st = take_wait_counter(dc, &n)) != MOBA_OK) return st;
    if (n != 0) return MOBA_ERR_HIP;
  }
  for (int g0 = 0; g0 < p.Hkv; g0 += nch) {
    a.g0 = g0;
    a.g1 = std::min(p.Hkv, g0 + nch);
    const int64_t e_chunk = pl->hist_per_head * p.G * (a.g1 - a.g0);
    if (routed && e_chunk > 0) {
      const int64_t grid = ceil_div(e_chunk, kTileRowsMfma) + (int64_t)(a.g1 - a.g0) * p.nblk_total;
      Phase ph("bwd_dq_hist", stream);
      MOBA_LAUNCH(launch_bwd_dq_hist(a, p, grid, stream));
    }
    Phase ph("bwd_dq_cur", stream);
    MOBA_LAUNCH(launch_bwd_dq_cur(a, p, stream));
  }
  return MOBA_OK;
}

}  // namespace

extern "C" {

moba_status moba_backward(const moba_tensor* q, const moba_tensor* k, const moba_tensor* v,
                          const moba_tensor* cu_seqlens, int32_t block_size, int32_t topk,
                          const moba_tensor* out, const moba_tensor* lse, const moba_tensor* dout,
                          moba_tensor* dq, moba_tensor* dk, moba_tensor* dv, hipStream_t stream) {
  return backward_impl(q, k, v, cu_seqlens, block_size, topk, out, lse, dout, dq, dk, dv, stream,
                       false);
}

moba_status moba_dense_backward(const moba_tensor* q, const moba_tensor* k, const moba_tensor* v,
                                const moba_tensor* cu_seqlens, const moba_tensor* out,
                                const moba_tensor* lse, const moba_tensor* dout, moba_tensor* dq,
                                moba_tensor* dk, moba_tensor* dv, hipStream_t stream) {
  return backward_impl(q, k, v, cu_seqlens, 0, 0, out, lse, dout, dq, dk, dv, stream, true);
}

moba_status moba_dense_forward(const moba_tensor* q, const moba_tensor* k, const moba_tensor* v,
                               const moba_tensor* cu_seqlens, moba_tensor* out, moba_tensor* lse,
                               hipStream_t stream) {
  Inputs in;
  View vo;
  moba_status st = check_inputs(q, k, v, cu_seqlens, out, lse, &in, &vo);
  if (st != MOBA_OK) return st;
  if ((st = read_cu(cu_seqlens, in.T, stream, &in.cu)) != MOBA_OK) return st;
  if (in.T == 0) return MOBA_OK;
  return dense_forward_impl(in, vo, lse, stream);
}

}  // extern "C"

namespace {

// Causal full attention over validated inputs (cu_seqlens already on the host).
moba_status dense_forward_impl(const Inputs& in, const View& vo, moba_tensor* lse,
                               hipStream_t stream) {
  moba_status st;
  std::lock_guard<std::mutex> lk(g_mu);
  DevCache* dc = cache_for_current_device();
  if (!dc) return MOBA_ERR_HIP;
  const Plan* pl;
  const SeqInfo* d_seqs;
  const CausalTile* d_tiles;
  if ((st = get_plan(dc, stream, in.cu, in.Hq, in.Hkv, 0, 1, kTilesDense,
                         in.bf16 ? kTileRowsMfma : kTileRowsF32, &pl, &d_seqs, &d_tiles)) != MOBA_OK)
    return st;
  const Problem& p = pl->p;
  Bump sz(nullptr);
  sz.take<__hip_bfloat16>(in.bf16 ? (int64_t)p.Hkv * p.vt_tiles * kKeyTile * kHeadDim : 0);
  if (sz.off + kAlign > workspace_limit()) return MOBA_ERR_NO_MEMORY;
  if ((st = ensure_workspace(dc, sz.off + kAlign)) != MOBA_OK) return st;
  Bump bp(dc->ws);
  AttnArgs a = make_args(in, vo, static_cast<float*>(lse->data));
  __hip_bfloat16* vt =
      bp.take<__hip_bfloat16>(in.bf16 ? (int64_t)p.Hkv * p.vt_tiles * kKeyTile * kHeadDim : 0);
  a.vt = vt;
  a.seqs = d_seqs;
  a.tiles = d_tiles;
  a.ntiles = (int64_t)pl->tiles.size();
  a.g0 = 0;
  a.g1 = p.Hkv;
  if (in.bf16) {
    Phase ph("vt_pack", stream);
    MOBA_LAUNCH(launch_vt_pack(static_cast<const __hip_bfloat16*>(in.v.data), in.v.st, in.v.sh,
                               d_seqs, p, vt, stream));
  }
  { Phase ph("dense", stream);
    MOBA_LAUNCH(in.bf16 ? launch_attn_causal_bf16(true, a, p, stream)
                        : launch_attn_causal_f32(true, a, p, stream)); }
  return MOBA_OK;
}

// moba_decode; with `noalloc`, moba_decode_noalloc: the per-shape tables are
// built on the host and written into the device's static scratch array by
// kernels that take them as arguments, and the buffers are carved from that
// array, so nothing is allocated.
moba_status decode_impl(const moba_tensor* q, const moba_tensor* k_cache,
                        const moba_tensor* v_cache, const moba_tensor* cu_seqlens,
                        const moba_tensor* kbar, int32_t block_size, int32_t topk, moba_tensor* out,
                        moba_tensor* lse, hipStream_t stream, bool noalloc) {
  if (missing(q) || missing(k_cache) || missing(v_cache) || missing(out) || missing(lse) ||
      !cu_seqlens || !cu_seqlens->data)
    return MOBA_ERR_NULL;
  if (q->dtype != MOBA_BF16) return MOBA_ERR_DTYPE;
  View vq, vk, vv, vo;
  moba_status st;
  if ((st = check_3d(q, MOBA_BF16, &vq)) != MOBA_OK) return st;
  if ((st = check_3d(k_cache, MOBA_BF16, &vk)) != MOBA_OK) return st;
  if ((st = check_3d(v_cache, MOBA_BF16, &vv)) != MOBA_OK) return st;
  if ((st = check_3d(out, MOBA_BF16, &vo)) != MOBA_OK) return st;
  const int64_t S = q->shape[0], T = k_cache->shape[0];
  const int Hq = (int)q->shape[1], Hkv = (int)k_cache->shape[1];
  if (v_cache->shape[0] != T || v_cache->shape[1] != Hkv || out->shape[0] != S ||
      out->shape[1] != Hq || Hq % Hkv != 0)
    return MOBA_ERR_SHAPE;
  if (Hq / Hkv > kDecodeMaxGroup) return MOBA_ERR_UNSUPPORTED;
  const int64_t lshape[2] = {Hq, S};
  if ((st = check_contig(lse, MOBA_F32, 2, lshape)) != MOBA_OK) return st;
  if ((st = check_cu_desc(cu_seqlens)) != MOBA_OK) return st;
  if (cu_seqlens->shape[0] != S + 1) return MOBA_ERR_SHAPE;
  if (topk < 0) return MOBA_ERR_TOPK;
  const bool want_full = topk == 0;
  if (!want_full && block_size < 1) return MOBA_ERR_BLOCK_SIZE;
  if (T >= (int64_t(1) << 31)) return MOBA_ERR_UNSUPPORTED;
  std::vector<int32_t> cu;
  if (noalloc && on_device(cu_seqlens->data)) return MOBA_ERR_UNSUPPORTED;
  if ((st = read_cu(cu_seqlens, T, stream, &cu)) != MOBA_OK) return st;
  if (S == 0) return MOBA_OK;
  int64_t lmax = 0;
  for (int64_t s = 0; s < S; s++) {
    if (cu[s + 1] == cu[s]) return MOBA_ERR_SEQLENS;  // every query needs its own cached token
    lmax = std::max<int64_t>(lmax, (int64_t)cu[s + 1] - cu[s]);
  }
  // top-k covering every block of every sequence is full attention
  const bool full = want_full || topk >= ceil_div(lmax, block_size);
  const int B = full ? kDecodeChunk : block_size;
  const int64_t nbmax = ceil_div(lmax, B);
  if (!full && nbmax > kMaxBlocksPerSeq) return MOBA_ERR_UNSUPPORTED;
  const int kk = full ? 1 : (int)std::min<int64_t>(topk, nbmax);
  if (kbar && !want_full) {
    if (missing(kbar)) return MOBA_ERR_NULL;
    int64_t nb = 0;
    for (int64_t s = 0; s < S; s++) nb += ceil_div((int64_t)cu[s + 1] - cu[s], block_size);
    const int64_t ks[3] = {nb, Hkv, kHeadDim};
    if ((st = check_contig(kbar, MOBA_F32, 3, ks)) != MOBA_OK) return st;
  }

  std::unique_lock<std::mutex> lk(g_mu, std::defer_lock);
  DevCache* dc = nullptr;
  const Plan* pl;
  Plan own_plan;
  const SeqInfo* d_seqs = nullptr;
  char* scratch_base = nullptr;
  if (noalloc) {
    if ((st = noalloc_scratch(&scratch_base)) != MOBA_OK) return st;
    build_plan(cu, Hkv, Hkv, B, kk, kTilesNone, kTileRowsMfma, &own_plan);
    pl = &own_plan;
  } else {
    lk.lock();
    dc = cache_for_current_device();
    if (!dc) return MOBA_ERR_HIP;
    const CausalTile* d_tiles;
    if ((st = get_plan(dc, stream, cu, Hkv, Hkv, B, kk, kTilesNone, kTileRowsMfma, &pl, &d_seqs,
                       &d_tiles)) != MOBA_OK)
      return st;
  }
  Problem p = pl->p;
  p.S = (int)S;
  p.Hq = Hq;
  p.G = Hq / Hkv;
  p.topk = kk;
  const int nsub = full ? 1 : (int)ceil_div(B, kDecodeChunk);
  const int64_t nchunk = nbmax * nsub;
  // blocks any head of a group can select: G (k - 1) history blocks plus the current one
  const int nunion = full ? 0 : (int)std::min<int64_t>(nbmax, (int64_t)(Hq / Hkv) * (kk - 1) + 1);
  const bool own_kbar = !full && !kbar;
  // combine: a row's partial slots (its chunks, or its selections' chunks)
  // in shares of kCombineShare, one work-group each
  const int64_t nslot = full ? nchunk : (int64_t)kk * nsub;
  const int nsplit = (int)std::min<int64_t>(kCombineMaxSplit, ceil_div(nslot, kCombineShare));
  const int split_len = (int)ceil_div(nslot, nsplit);
  auto layout = [&](Bump* bp, float** kb, int32_t** sel, float** po, float** pls, float** mid) {
    if (noalloc) d_seqs = bp->take<SeqInfo>(S);  // the tables, first
    *kb = bp->take<float>(own_kbar ? (int64_t)p.nblk_total * Hkv * kHeadDim : 0);
    *sel = bp->take<int32_t>(full ? 0 : S * Hq * kk);
    *po = bp->take<float>(S * Hq * nchunk * kHeadDim);
    *pls = bp->take<float>(S * Hq * nchunk);
    *mid = bp->take<float>(nsplit > 1 ? S * Hq * nsplit * (kHeadDim + 2) : 0);
  };
  {
    Bump sz(nullptr);
    float *a0, *a2, *a3, *a5;
    int32_t* a1;
    layout(&sz, &a0, &a1, &a2, &a3, &a5);
    if (noalloc) {
      if (sz.off > kNoAllocScratchBytes) return MOBA_ERR_NO_MEMORY;
    } else {
      if (sz.off + kAlign > workspace_limit()) return MOBA_ERR_NO_MEMORY;
      if ((st = ensure_workspace(dc, sz.off + kAlign)) != MOBA_OK) return st;
    }
  }
  Bump bp(noalloc ? static_cast<void*>(scratch_base) : dc->ws);
  DecodeArgs a{};
  float* kb_ws;
  layout(&bp, &kb_ws, &a.sel, &a.part_o, &a.part_lse, &a.mid);
  if (noalloc) {
    // the per-sequence table, written by kernels that receive it by value
    SeqInfo* dst = const_cast<SeqInfo*>(d_seqs);
    for (int64_t s0 = 0; s0 < S; s0 += kSeqsPerCopy) {
      SeqBatch b{};
      b.n = (int32_t)std::min<int64_t>(kSeqsPerCopy, S - s0);
      for (int i = 0; i < b.n; i++) b.s[i] = pl->seqs[s0 + i];
      MOBA_LAUNCH(launch_seq_table(b, dst + s0, stream));
    }
  }
  a.nsplit = nsplit;
  a.split_len = split_len;
  a.nunion = nunion;
  a.q = static_cast<const __hip_bfloat16*>(vq.data); a.q_ss = vq.st; a.q_sh = vq.sh;
  a.k = static_cast<const __hip_bfloat16*>(vk.data); a.k_st = vk.st; a.k_sh = vk.sh;
  a.v = static_cast<const __hip_bfloat16*>(vv.data); a.v_st = vv.st; a.v_sh = vv.sh;
  a.out = static_cast<__hip_bfloat16*>(vo.data); a.o_ss = vo.st; a.o_sh = vo.sh;
  a.lse = static_cast<float*>(lse->data);
  a.kbar = own_kbar ? kb_ws : (full ? nullptr : static_cast<const float*>(kbar->data));
  a.seqs = d_seqs;
  a.nsub = nsub;
  a.nchunk = (int)nchunk;
  a.chunk_block = B;
  a.full = full ? 1 : 0;
  a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)kHeadDim));
  // (the no-alloc path records no profiling events)
  if (own_kbar) {
    Phase ph(noalloc ? nullptr : "pool", stream);
    MOBA_LAUNCH(launch_pool(vk.data, true, vk.st, vk.sh, d_seqs, p, kb_ws, nullptr, stream));
  }
  if (!full) {
    Phase ph(noalloc ? nullptr : "decode_gate", stream);
    MOBA_LAUNCH(launch_decode_gate(a, p, stream));
  }
  { Phase ph(noalloc ? nullptr : "decode_attend", stream);
    MOBA_LAUNCH(launch_decode_attend(a, p, stream)); }
  { Phase ph(noalloc ? nullptr : "decode_combine", stream);
    MOBA_LAUNCH(launch_decode_combine(a, p, stream)); }
  return MOBA_OK;
}


}  // namespace

extern "C" {

moba_status moba_decode(const moba_tensor* q, const moba_tensor* k_cache,
                        const moba_tensor* v_cache, const moba_tensor* cu_seqlens,
                        const moba_tensor* kbar, int32_t block_size, int32_t topk, moba_tensor* out,
                        moba_tensor* lse, hipStream_t stream) {
  return decode_impl(q, k_cache, v_cache, cu_seqlens, kbar, block_size, topk, out, lse, stream,
                     false);
}

moba_status moba_decode_noalloc(const moba_tensor* q, const moba_tensor* k_cache,
                                const moba_tensor* v_cache, const moba_tensor* cu_seqlens,
                                const moba_tensor* kbar, int32_t block_size, int32_t topk,
                                moba_tensor* out, moba_tensor* lse, hipStream_t stream) {
  return decode_impl(q, k_cache, v_cache, cu_seqlens, kbar, block_size, topk, out, lse, stream,
                     true);
}

moba_status moba_pool(const moba_tensor* k, const moba_tensor* cu_seqlens, int32_t block_size,
                      moba_tensor* kbar, hipStream_t stream) {
  if (missing(k) || missing(kbar) || !cu_seqlens || !cu_seqlens->data) return MOBA_ERR_NULL;
  if (k->dtype != MOBA_BF16 && k->dtype != MOBA_F32) return MOBA_ERR_DTYPE;
  View vk;
  moba_status st = check_3d(k, k->dtype, &vk);
  if (st != MOBA_OK) return st;
  if ((st = check_cu_desc(cu_seqlens)) != MOBA_OK) return st;
  if (block_size < 1) return MOBA_ERR_BLOCK_SIZE;
  std::vector<int32_t> cu;
  if ((st = read_cu(cu_seqlens, k->shape[0], stream, &cu)) != MOBA_OK) return st;
  const int Hkv = (int)k->shape[1];
  int64_t nb = 0;
  for (size_t s = 0; s + 1 < cu.size(); s++) nb += ceil_div((int64_t)cu[s + 1] - cu[s], block_size);
  const int64_t shp[3] = {nb, Hkv, kHeadDim};
  if ((st = check_contig(kbar, MOBA_F32, 3, shp)) != MOBA_OK) return st;
  if (nb == 0) return MOBA_OK;
  std::lock_guard<std::mutex> lk(g_mu);
  DevCache* dc = cache_for_current_device();
  if (!dc) return MOBA_ERR_HIP;
  const Plan* pl;
  const SeqInfo* d_seqs;
  const CausalTile* d_tiles;
  if ((st = get_plan(dc, stream, cu, Hkv, Hkv, block_size, 1, kTilesNone, kTileRowsMfma, &pl, &d_seqs,
                      &d_tiles)) != MOBA_OK)
    return st;
  Phase ph("pool", stream);
  MOBA_LAUNCH(launch_pool(vk.data, k->dtype == MOBA_BF16, vk.st, vk.sh, d_seqs, pl->p,
                          static_cast<float*>(kbar->data), nullptr, stream));
  return MOBA_OK;
}

moba_status moba_select(const moba_tensor* q, const moba_tensor* k, const moba_tensor* cu_seqlens,
                        int32_t block_size, int32_t topk, moba_tensor* sel, moba_tensor* scores,
                        hipStream_t stream) {
  if (missing(q) || missing(k) || missing(sel) || !cu_seqlens || !cu_seqlens->data)
    return MOBA_ERR_NULL;
  if (q->dtype != MOBA_BF16 && q->dtype != MOBA_F32) return MOBA_ERR_DTYPE;
  View vq, vk;
  moba_status st;
  if ((st = check_3d(q, q->dtype, &vq)) != MOBA_OK) return st;
  if ((st = check_3d(k, q->dtype, &vk)) != MOBA_OK) return st;
  const int64_t T = q->shape[0];
  const int Hq = (int)q->shape[1], Hkv = (int)k->shape[1];
  if (k->shape[0] != T || Hq % Hkv != 0) return MOBA_ERR_SHAPE;
  if (Hq / Hkv > kMaxGroup) return MOBA_ERR_UNSUPPORTED;
  if ((st = check_cu_desc(cu_seqlens)) != MOBA_OK) return st;
  if (block_size < 1) return MOBA_ERR_BLOCK_SIZE;
  if (topk < 1) return MOBA_ERR_TOPK;
  const int64_t sshape[3] = {T, Hq, topk};
  if ((st = check_contig(sel, MOBA_I32, 3, sshape)) != MOBA_OK) return st;
  int nmax = 0;
  if (scores) {
    if (missing(scores)) return MOBA_ERR_NULL;
    if (scores->ndim != 3) return MOBA_ERR_SHAPE;
    const int64_t scs[3] = {T, Hq, scores->shape[2]};
    if (scores->shape[2] < 1 || scores->shape[2] > (1 << 20)) return MOBA_ERR_SHAPE;
    if ((st = check_contig(scores, MOBA_F32, 3, scs)) != MOBA_OK) return st;
    nmax = (int)scores->shape[2];
  }
  std::vector<int32_t> cu;
  if ((st = read_cu(cu_seqlens, T, stream, &cu)) != MOBA_OK) return st;
  if (T == 0) return MOBA_OK;
  int64_t nbmax = 0;
  for (size_t s = 0; s + 1 < cu.size(); s++)
    nbmax = std::max<int64_t>(nbmax, ceil_div((int64_t)cu[s + 1] - cu[s], block_size));
  if (topk - 1 > 63 && topk - 1 < nbmax - 1) return MOBA_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lk(g_mu);
  DevCache* dc = cache_for_current_device();
  if (!dc) return MOBA_ERR_HIP;
  const Plan* pl;
  const SeqInfo* d_seqs;
  const CausalTile* d_tiles;
  if ((st = get_plan(dc, stream, cu, Hq, Hkv, block_size, topk, kTilesNone, kTileRowsMfma, &pl, &d_seqs,
                      &d_tiles)) != MOBA_OK)
    return st;
  const Problem& p = pl->p;
  const bool bf16 = q->dtype == MOBA_BF16;
  const int64_t nkb = (int64_t)p.nblk_total * Hkv * kHeadDim;
  Bump sz(nullptr);
  sz.take<float>(nkb);
  sz.take<__hip_bfloat16>(bf16 ? 3 * nkb : 0);
  if (sz.off + kAlign > workspace_limit()) return MOBA_ERR_NO_MEMORY;
  if ((st = ensure_workspace(dc, sz.off + kAlign)) != MOBA_OK) return st;
  Bump bp(dc->ws);
  float* kbar = bp.take<float>(nkb);
  __hip_bfloat16* kterm = bf16 ? bp.take<__hip_bfloat16>(3 * nkb) : nullptr;
  { Phase ph("pool", stream);
    MOBA_LAUNCH(launch_pool(vk.data, bf16, vk.st, vk.sh, d_seqs, p, kbar, kterm, stream)); }
  { Phase ph("gate", stream);
    MOBA_LAUNCH(launch_gate(vq.data, bf16, vq.st, vq.sh, kbar, kterm, d_seqs, p,
                            static_cast<int32_t*>(sel->data),
                            scores ? static_cast<float*>(scores->data) : nullptr, nmax, stream)); }
  return MOBA_OK;
}

moba_status moba_route(const moba_tensor* sel, const moba_tensor* cu_seqlens, int32_t block_size,
                       int32_t num_kv_heads, moba_tensor* counts, moba_tensor* offsets,
                       moba_tensor* entries, hipStream_t stream) {
  if (missing(sel) || !cu_seqlens || !cu_seqlens->data || missing(counts) || missing(offsets) ||
      !entries)
    return MOBA_ERR_NULL;
  if (sel->dtype != MOBA_I32) return MOBA_ERR_DTYPE;
  if (sel->ndim != 3) return MOBA_ERR_SHAPE;
  const int64_t T = sel->shape[0];
  const int Hq = (int)sel->shape[1];
  const int topk = (int)sel->shape[2];
  const int64_t ss[3] = {T, Hq, topk};
  moba_status st;
  if ((st = check_contig(sel, MOBA_I32, 3, ss)) != MOBA_OK) return st;
  if (num_kv_heads < 1 || Hq < 1 || Hq % num_kv_heads != 0) return MOBA_ERR_SHAPE;
  if (Hq / num_kv_heads > kMaxGroup) return MOBA_ERR_UNSUPPORTED;
  if (block_size < 1) return MOBA_ERR_BLOCK_SIZE;
  if (topk < 1) return MOBA_ERR_TOPK;
  if ((st = check_cu_desc(cu_seqlens)) != MOBA_OK) return st;
  std::vector<int32_t> cu;
  if ((st = read_cu(cu_seqlens, T, stream, &cu)) != MOBA_OK) return st;
  int64_t nbmax = 0, nb = 0;
  for (size_t s = 0; s + 1 < cu.size(); s++) {
    const int64_t n = ceil_div((int64_t)cu[s + 1] - cu[s], block_size);
    nbmax = std::max(nbmax, n);
    nb += n;
  }
  if (nbmax > kMaxBlocksPerSeq) return MOBA_ERR_UNSUPPORTED;
  if ((uint64_t)T * Hq * (uint64_t)std::max(topk - 1, 1) >= (uint64_t(1) << 32))
    return MOBA_ERR_UNSUPPORTED;
  const int64_t nbins = nb * num_kv_heads;
  const int64_t cs[1] = {nbins};
  const int64_t os[1] = {nbins + 1};
  if ((st = check_contig(counts, MOBA_I32, 1, cs)) != MOBA_OK) return st;
  if ((st = check_contig(offsets, MOBA_I64, 1, os)) != MOBA_OK) return st;
  std::lock_guard<std::mutex> lk(g_mu);
  DevCache* dc = cache_for_current_device();
  if (!dc) return MOBA_ERR_HIP;
  const Plan* pl;
  const SeqInfo* d_seqs;
  const CausalTile* d_tiles;
  if ((st = get_plan(dc, stream, cu, Hq, num_kv_heads, block_size, topk, kTilesNone, kTileRowsMfma, &pl,
                     &d_seqs, &d_tiles)) != MOBA_OK)
    return st;
  const Problem& p = pl->p;
  const int64_t es[1] = {p.hist_entries};
  if (p.hist_entries > 0) {
    if (missing(entries)) return MOBA_ERR_NULL;
    if ((st = check_contig(entries, MOBA_I32, 1, es)) != MOBA_OK) return st;
  } else if (entries->ndim != 1 || entries->shape[0] != 0) {
    return MOBA_ERR_SHAPE;
  }
  if (nbins == 0) return MOBA_OK;
  Bump sz(nullptr);
  sz.take<int32_t>((int64_t)p.Hkv * p.hist_words);
  sz.take<int32_t>(nbins + 1);
  if (sz.off + kAlign > workspace_limit()) return MOBA_ERR_NO_MEMORY;
  if ((st = ensure_workspace(dc, sz.off + kAlign)) != MOBA_OK) return st;
  Bump bp(dc->ws);
  RouteBuffers rb{};
  rb.hist = bp.take<int32_t>((int64_t)p.Hkv * p.hist_words);
  rb.bin_tile_start = bp.take<int32_t>(nbins + 1);
  rb.bin_count = static_cast<int32_t*>(counts->data);
  rb.bin_start = static_cast<int64_t*>(offsets->data);
  rb.entries = static_cast<uint32_t*>(entries->data);
  Phase ph("route", stream);
  MOBA_LAUNCH(launch_route(static_cast<const int32_t*>(sel->data), d_seqs, p, rb, stream));
  return MOBA_OK;
}

size_t moba_workspace_bytes(int64_t T, int32_t Hq, int32_t Hkv, int32_t D, int64_t nblk_total,
                            int32_t topk) {
  if (T < 0 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || Hq / Hkv > kMaxGroup || D != kHeadDim ||
      nblk_total < 0 || topk < 1)
    return 0;
  if (T == 0 || nblk_total == 0) return 0;
  // bounds over every cu_seqlens with these totals (each non-empty sequence
  // holds at least one block, and no sequence more than nblk_total)
  Problem p{};
  p.T = T;
  p.Hq = Hq;
  p.Hkv = Hkv;
  p.G = Hq / Hkv;
  p.nblk_total = (int)std::min<int64_t>(nblk_total, INT32_MAX);
  p.vt_tiles = ceil_div(T, kKeyTile) + nblk_total;
  p.tile_rows = std::min(kTileRowsMfma, kTileRowsF32);  // the smaller gives more tiles
  const int kk = (int)std::min<int64_t>(topk, nblk_total);
  p.hist_words = (ceil_div(T, std::max(1, kRouteRows / p.G)) + 1) * nblk_total;
  p.hist_entries = T * Hq * (int64_t)(kk - 1);
  size_t need = 0;
  for (int bf16 = 0; bf16 < 2; bf16++) {
    Bump bp(nullptr);
    FwdBufs b{};
    forward_layout(p, bf16 != 0, kk, Hkv, &bp, &b);
    need = std::max(need, bp.off + kAlign);
  }
  return need;
}

moba_status moba_route_size(const moba_tensor* cu_seqlens, int32_t block_size, int32_t topk,
                            int32_t num_q_heads, int64_t* nblk_total, int64_t* entries,
                            hipStream_t stream) {
  if (!nblk_total || !entries) return MOBA_ERR_NULL;
  moba_status st;
  if ((st = check_cu_desc(cu_seqlens)) != MOBA_OK) return st;
  if (block_size < 1) return MOBA_ERR_BLOCK_SIZE;
  if (topk < 1) return MOBA_ERR_TOPK;
  if (num_q_heads < 1) return MOBA_ERR_SHAPE;
  std::vector<int32_t> cu;
  if ((st = fetch_cu(cu_seqlens, stream, &cu)) != MOBA_OK) return st;
  if ((st = check_cu(cu, cu.back())) != MOBA_OK) return st;  // the batch holds T = cu[S] tokens
  batch_sizes(cu, block_size, topk, num_q_heads, nblk_total, entries);
  return MOBA_OK;
}

moba_status moba_take_wait_timeouts(uint64_t* count) {
  if (!count) return MOBA_ERR_NULL;
  std::lock_guard<std::mutex> lk(g_mu);
  DevCache* dc = cache_for_current_device();
  if (!dc) return MOBA_ERR_HIP;
  return take_wait_counter(dc, count);
}

size_t moba_workspace_held_bytes(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  auto it = g_dev.find(dev);
  return it == g_dev.end() ? 0 : it->second.ws_bytes;
}

moba_status moba_release_workspace(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MOBA_ERR_HIP;
  auto it = g_dev.find(dev);
  if (it == g_dev.end()) return MOBA_OK;
  if (hipDeviceSynchronize() != hipSuccess) return MOBA_ERR_HIP;
  if (it->second.ws) (void)hipFree(it->second.ws);
  if (it->second.wait_timeouts) (void)hipFree(it->second.wait_timeouts);
  for (PlanSlot& sl : it->second.slots) {
    if (sl.tab) (void)hipFree(sl.tab);
    if (sl.stage) (void)hipHostFree(sl.stage);
    if (sl.uploaded) (void)hipEventDestroy(sl.uploaded);
  }
  g_dev.erase(it);
  return MOBA_OK;
}

const char* moba_status_string(moba_status s) {
  switch (s) {
    case MOBA_OK: return "MOBA_OK";
    case MOBA_ERR_NULL: return "MOBA_ERR_NULL";
    case MOBA_ERR_DTYPE: return "MOBA_ERR_DTYPE";
    case MOBA_ERR_SHAPE: return "MOBA_ERR_SHAPE";
    case MOBA_ERR_LAYOUT: return "MOBA_ERR_LAYOUT";
    case MOBA_ERR_BLOCK_SIZE: return "MOBA_ERR_BLOCK_SIZE";
    case MOBA_ERR_TOPK: return "MOBA_ERR_TOPK";
    case MOBA_ERR_SEQLENS: return "MOBA_ERR_SEQLENS";
    case MOBA_ERR_UNSUPPORTED: return "MOBA_ERR_UNSUPPORTED";
    case MOBA_ERR_NO_MEMORY: return "MOBA_ERR_NO_MEMORY";
    case MOBA_ERR_HIP: return "MOBA_ERR_HIP";
  }
  return "MOBA_ERR_UNKNOWN";
}

void moba_profile_enable(int enabled) { g_prof = enabled != 0; }

int moba_profile_read(moba_phase_stat* stats, int max_phases) {
  std::vector<PhaseRec> recs;
  {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    recs.swap(g_recs);
  }
  std::vector<moba_phase_stat> acc;
  for (const PhaseRec& r : recs) {
    float ms = 0.0f;
    if (hipEventSynchronize(r.b) == hipSuccess && hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess) {
      auto it = std::find_if(acc.begin(), acc.end(),
                             [&](const moba_phase_stat& x) { return std::strcmp(x.name, r.name) == 0; });
      if (it == acc.end()) {
        moba_phase_stat z{};
        std::strncpy(z.name, r.name, sizeof(z.name) - 1);
        acc.push_back(z);
        it = acc.end() - 1;
      }
      it->launches += 1;
      it->total_ms += ms;
    }
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  const int n = std::min<int>((int)acc.size(), std::max(max_phases, 0));
  for (int i = 0; i < n; i++) stats[i] = acc[i];
  return n;
}

}  // extern "C"
