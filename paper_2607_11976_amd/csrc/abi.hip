// C ABI of the library (include/litetopk.h): argument checks, option
// resolution, workspace carving and the stream-ordered launch sequence.
#include <string.h>

#include <algorithm>
#include <mutex>

#include "internal.hpp"
#include "select_dev.hpp"

using namespace lt;

// Workspace of lt_indexer_topk_static: one copy per GPU, held until the
// process ends. In host code `scratch` names a host-side stand-in, never the
// device memory: host code uses only the address hipGetSymbolAddress returns
// for the current device (static_scratch below).
static __device__ __align__(256) uint8_t scratch[LT_STATIC_SCRATCH_BYTES];

namespace {

constexpr int kDefaultBins = 256;
constexpr size_t kFallbackScratchBudget = 2ull << 30;  // bytes of scratch the dense fallback may take
// blocks of the scores-in fallback: one per row up to 2048 rows (several
// resident per CU hide the radix select's load latency), at least 256
constexpr int kFallbackGridScoresMin = 256, kFallbackGridScoresMax = 2048;
constexpr int kTargetBlocks = 256;          // one block per CU before key splitting stops
constexpr int kMinSplitKeys = 512;          // shortest key split the automatic choice makes
constexpr int kMaxAutoSplits = 64;
constexpr size_t kHistLdsBudget = 96 * 1024;
constexpr size_t kLdsPerBlock = 160 * 1024;   // gfx950 LDS per workgroup
constexpr int kSampleBlockScores = 64;      // scores-in sample: runs of 64 consecutive keys
constexpr int kMinSharedSplitKeys = 1024;   // shortest key split of the shared-row (wide) scan
constexpr int kSharedSample = 65536;        // default sample of the shared-row scan (inner product)

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct Resolved {
  int k, m, ns, cap, S, L, E;
  int HS;                  // histograms per row: S, or 1 when shared by the splits
  bool shared;             // the wide scan: one histogram and threshold per row
  uint32_t flags;
  uint64_t seed;
  void** ev;
  int32_t* stats;
  const int32_t* keys_in;  // caller's sample list, or NULL for the random sample
  const int32_t* starts;   // per-row visible starts, or NULL
  int status;              // LT_OK, or the error the options produce
};

struct Layout {
  size_t qctl, queue, rqueue, rflag, params, list, samp, cnt, hist, cand, gate, scratch, fbcand, total;
};

// The dense fallback's scratch, in fp32 rows of Nk scores: in whole-row mode
// `grid` blocks re-score `batch` rows of one query tile per pass, each into
// its own scratch rows. Up to kFallbackGrid rows: one row per block. More
// rows: kFallbackGrid blocks, each taking up to kMaxFallbackBatch rows of a
// tile per pass, so that a tile whose rows all fall back is scored once or
// twice instead of once per row. Within the scratch budget: fewer rows per
// pass, then fewer blocks (down to 64). Split mode (few queued rows, each
// row's keys over many blocks) takes one of the same rows per queued row.
struct FallbackShape {
  int grid, batch;
};
FallbackShape fallback_shape(int nq, int nk) {
  const size_t row = (size_t)std::max(nk, 1) * 4;
  FallbackShape f{std::max(1, std::min(nq, kFallbackGrid)), 1};
  if (nq > kFallbackGrid) f.batch = std::min(kMaxFallbackBatch, (nq + kFallbackGrid - 1) / kFallbackGrid);
  if ((size_t)f.grid * f.batch * row > kFallbackScratchBudget)
    f.batch = (int)std::max<size_t>(1, kFallbackScratchBudget / ((size_t)f.grid * row));
  if ((size_t)f.grid * f.batch * row > kFallbackScratchBudget)
    f.grid = (int)std::max<size_t>(std::min(f.grid, 64), kFallbackScratchBudget / row);
  return f;
}

Layout carve(int nq, int nk, const Resolved& r, bool fused) {
  Layout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align256(off + bytes);
    return o;
  };
  L.qctl = take((size_t)kQctlWords * 4);
  L.queue = take((size_t)nq * 4);
  L.rqueue = fused ? take((size_t)nq * 4) : 0;  // rows of the second filter pass
  L.rflag = fused ? take((size_t)nq * 8) : 0;  // second-pass flags [nq], then dense-fallback flags [nq]
  L.params = take((size_t)nq * sizeof(RowParam));
  L.list = take((size_t)r.ns * 4);
  L.samp = fused ? take((size_t)nq * r.ns * 4) : 0;
  L.cnt = take((size_t)nq * r.S * 4);
  L.hist = take((size_t)nq * r.HS * r.m * 4);
  L.cand = take((size_t)nq * r.S * r.cap * 8);
  L.gate = fused ? take((size_t)nq * 8) : 0;  // published bins: [nq] ints (wide), [nq][8] bytes
  const FallbackShape fs = fallback_shape(nq, nk);
  L.scratch = fused ? take((size_t)fs.grid * fs.batch * nk * 4) : 0;
  // split fallback (both entries): the chunks' top-k candidates, (index,
  // score) arrays of kFallbackGrid * k entries each
  L.fbcand = take((size_t)kFallbackGrid * r.k * 8);
  L.total = off;
  return L;
}

int select_entries(int k) {
  int e = 2 * next_pow2(k);
  return e < 4096 ? 4096 : e;
}

// Options common to both filter pipelines.
void resolve_common(const lt_options* o, int k, Resolved& r) {
  lt_options d;
  lt_options_default(&d);
  if (!o) o = &d;
  r.m = o->num_bins > 0 ? std::min(o->num_bins, LT_MAX_BINS) : kDefaultBins;
  r.cap = o->capacity > 0 ? o->capacity : std::max(12 * k, 2048);
  r.flags = o->flags & (LT_SORTED_OUTPUT | LT_FORCE_FALLBACK);
  r.seed = o->seed;
  r.ev = o->stage_events;
  r.stats = o->row_stats;
  r.k = k;
  r.E = select_entries(k);
  r.shared = false;
  r.keys_in = o->sample_keys;
  r.starts = o->visible_start;
  r.status = LT_OK;
  if (r.keys_in && (o->sample_size < 1 || o->sample_size > LT_SAMPLE_LIST_MAX)) r.status = LT_EINVAL;
}

// Sample size: the caller's list length, or k' from the options and mode.
int resolve_sample(const lt_options* o, const Resolved& r, int nk, int k, int mode, bool fused) {
  if (r.keys_in) return r.status == LT_OK ? o->sample_size : 0;
  int ns = o->sample_size;
  if (ns < 0) {
    ns = 3 * k;  // sec. 3.2: k' = 3k
    if (fused && mode == LT_SCORE_IP) {
      // a random sample's k-th score sits at rank k * nk / ns of the corpus,
      // and the first tiles of every split run at that rank: the wide scan
      // samples kSharedSample keys, the grouped one nk / 128 (the 10000 x 4M
      // retrieval: nk / 64 took 15.9 ms a call, nk / 128 15.2, nk / 256 15.4;
      // its scoring and range stages grow with the sample, its survivors
      // shrink)
      ns = std::max(ns, r.shared ? kSharedSample : std::min(nk / 128, 65536));
    }
  }
  return sample_count(ns, nk);
}

Resolved resolve_fused(const lt_options* o, int nq, int nk, int k, int mode, const ScoreShape& sh) {
  Resolved r{};
  resolve_common(o, k, r);
  lt_options d;
  lt_options_default(&d);
  if (!o) o = &d;
  r.shared = sh.shared_rows != 0;
  // per-row LDS histograms share the block's LDS with the scan's own data
  const size_t room = kLdsPerBlock - sh.scan_lds - 64;
  const size_t mcap = std::min(kHistLdsBudget, room) / (4 * (size_t)sh.queries_per_block);
  if ((size_t)r.m > mcap) r.m = (int)std::max<size_t>(mcap, 1);
  if (r.shared && o->capacity <= 0) {
    // a split's list holds its share of the row's candidates (an online top-k
    // over N keys admits about k (1 + ln(N / k)), spread over the splits)
    // plus what the sample's threshold lets through before the first
    // refreshes; k more keeps a row whose whole top-k lies in one split
    r.cap = k + std::max(1024, k / 2);
  }
  // the shared scan's lists are stored in chunks of 16 entries
  if (r.shared) r.cap = (r.cap + 15) & ~15;
  r.ns = resolve_sample(o, r, nk, k, mode, true);
  const int steps = (nk + sh.keys_per_step - 1) / sh.keys_per_step;
  const int tiles = (nq + sh.queries_per_block - 1) / sh.queries_per_block;
  int S = 1;
  if (o->key_splits > 0) {
    S = std::min(o->key_splits, std::max(steps, 1));
  } else if (r.shared) {
    // the splits share their thresholds, so splitting costs no survivors:
    // enough blocks for one per CU, each split keeping kMinSharedSplitKeys
    S = std::max(1, std::min((kTargetBlocks + tiles - 1) / tiles, nk / kMinSharedSplitKeys));
  } else {
    // The fewest key splits whose launch keeps at least 90% of the block
    // slots busy in its last round (one block per CU), each split keeping at
    // least kMinSplitKeys keys. Each split tightens its threshold only from
    // its own histogram, so a split adds survivors when the initial threshold
    // is loose; a launch that leaves most CUs idle loses far more.
    const int smax = std::max(1, std::min(kMaxAutoSplits, nk / kMinSplitKeys));
    for (int s = 1; s <= smax; ++s) {
      const long long blocks = (long long)tiles * s;
      const long long rounds = (blocks + kTargetBlocks - 1) / kTargetBlocks;
      S = s;
      if (blocks * 10 >= rounds * kTargetBlocks * 9) break;
    }
  }
  r.S = S;
  r.HS = r.shared ? 1 : S;
  const int per = (nk + S - 1) / S;
  r.L = ((per + sh.keys_per_step - 1) / sh.keys_per_step) * sh.keys_per_step;
  if (r.L == 0) r.L = sh.keys_per_step;
  return r;
}

Resolved resolve_scores(const lt_options* o, int nq, int nk, int k) {
  Resolved r{};
  resolve_common(o, k, r);
  lt_options d;
  lt_options_default(&d);
  if (!o) o = &d;
  r.ns = resolve_sample(o, r, nk, k, LT_SCORE_DSA, false);
  int S = 1;
  if (o->key_splits > 0) S = o->key_splits;
  r.S = std::max(1, std::min(S, (nk + 255) / 256 + 1));
  r.HS = r.S;
  const int per = (nk + r.S - 1) / r.S;
  r.L = std::max(256, ((per + 255) / 256) * 256);
  (void)nq;
  return r;
}

inline bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

inline int hip_status(hipError_t e) { return e == hipSuccess ? LT_OK : LT_EHIP; }

// The launch's sample list: the caller's, cleaned, or the random one.
hipError_t make_list(const Resolved& r, int nk, int blk, int32_t* list, hipStream_t st) {
  if (r.keys_in) return launch_list_clean(r.keys_in, r.ns, nk, list, st);
  return launch_sample_list(list, r.ns, nk, blk, r.seed, st);
}

inline void record(const Resolved& r, int i, hipStream_t st) {
  if (r.ev && r.ev[i]) (void)hipEventRecord((hipEvent_t)r.ev[i], st);
}

int check_score_args(const void* q, const float* q_scale, const void* keys, const float* k_scale,
                     lt_dtype dtype, lt_score_mode mode, int nq, int nk, int h, int d) {
  if (nq < 0 || nk < 0 || h <= 0 || d <= 0) return LT_EINVAL;
  if (dtype != LT_F32 && dtype != LT_BF16 && dtype != LT_FP8_E4M3FN) return LT_EINVAL;
  if (mode != LT_SCORE_DSA && mode != LT_SCORE_IP) return LT_EINVAL;
  if (nq > 0 && (!q || !aligned(q, 16))) return LT_EINVAL;
  if (nk > 0 && (!keys || !aligned(keys, 16))) return LT_EINVAL;
  if (dtype == LT_FP8_E4M3FN && ((nq > 0 && !q_scale) || (nk > 0 && !k_scale))) return LT_EINVAL;
  if (!score_shape(dtype, mode, h, d).supported) return LT_EUNSUPPORTED;
  return LT_OK;
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // device address of `scratch`, per device

// This device's copy of `scratch`: looked up once per device, with that
// device current, on the first call made there.
int static_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return LT_EHIP;
  if (dev < 0 || dev >= kMaxDevices) return LT_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return LT_EHIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return LT_OK;
}

}  // namespace

extern "C" {

void lt_options_default(lt_options* o) {
  if (!o) return;
  memset(o, 0, sizeof(*o));
  o->num_bins = kDefaultBins;
  o->sample_size = -1;
  o->capacity = 0;
  o->key_splits = 0;
  o->flags = 0;
  o->seed = 0x5EED5EEDull;
  o->stage_events = nullptr;
  o->row_stats = nullptr;
  o->sample_keys = nullptr;
  o->visible_start = nullptr;
}

const char* lt_strerror(int status) {
  switch (status) {
    case LT_OK: return "ok";
    case LT_EINVAL: return "invalid argument";
    case LT_EUNSUPPORTED: return "unsupported (dtype, heads, head_dim, mode) or k";
    case LT_EWORKSPACE: return "workspace too small";
    case LT_EHIP: return "HIP runtime error";
    case LT_ESCRATCH: return "shape needs more workspace than the static scratch (LT_STATIC_SCRATCH_BYTES)";
    default: return "unknown status";
  }
}

size_t lt_indexer_topk_workspace_size(int32_t nq, int32_t nk, int32_t h, int32_t d, lt_dtype dtype,
                                      lt_score_mode mode, int32_t k, const lt_options* opts) {
  if (nq < 0 || nk < 0 || k < 1 || k > LT_K_MAX) return 0;
  ScoreShape sh = score_shape(dtype, mode, h, d);
  if (!sh.supported) return 0;
  Resolved r = resolve_fused(opts, nq, nk, k, mode, sh);
  if (r.status) return 0;
  return carve(nq, nk, r, true).total;
}

int lt_indexer_topk(const void* q, const float* q_scale, const float* w, const void* keys,
                    const float* k_scale, lt_dtype dtype, lt_score_mode mode, int32_t nq, int32_t nk,
                    int32_t h, int32_t d, int32_t k, const int32_t* offs, int32_t* out_idx,
                    float* out_scores, void* workspace, size_t workspace_bytes, const lt_options* opts,
                    void* stream) {
  int rc = check_score_args(q, q_scale, keys, k_scale, dtype, mode, nq, nk, h, d);
  if (rc) return rc;
  if (k < 1) return LT_EINVAL;
  if (k > LT_K_MAX) return LT_EUNSUPPORTED;
  if (nq == 0) return LT_OK;
  if (!out_idx || !out_scores || !workspace || !aligned(workspace, 256)) return LT_EINVAL;
  const ScoreShape sh = score_shape(dtype, mode, h, d);
  const Resolved r = resolve_fused(opts, nq, nk, k, mode, sh);
  if (r.status) return r.status;
  const Layout L = carve(nq, nk, r, true);
  if (workspace_bytes < L.total) return LT_EWORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  uint32_t* qctl = reinterpret_cast<uint32_t*>(ws + L.qctl);
  int32_t* queue = reinterpret_cast<int32_t*>(ws + L.queue);
  RowParam* params = reinterpret_cast<RowParam*>(ws + L.params);
  int32_t* list = reinterpret_cast<int32_t*>(ws + L.list);
  float* samp = reinterpret_cast<float*>(ws + L.samp);
  uint32_t* cnt = reinterpret_cast<uint32_t*>(ws + L.cnt);
  uint32_t* hist = reinterpret_cast<uint32_t*>(ws + L.hist);
  int2* cand = reinterpret_cast<int2*>(ws + L.cand);
  float* scratch = reinterpret_cast<float*>(ws + L.scratch);
  int32_t* fbc_idx = reinterpret_cast<int32_t*>(ws + L.fbcand);
  float* fbc_score = reinterpret_cast<float*>(ws + L.fbcand + (size_t)kFallbackGrid * k * 4);
  int* gate = reinterpret_cast<int*>(ws + L.gate);
  int32_t* rqueue = reinterpret_cast<int32_t*>(ws + L.rqueue);
  int32_t* rflag = reinterpret_cast<int32_t*>(ws + L.rflag);
  ScoreArgs a{q, q_scale, w, keys, k_scale, (int)dtype, (int)mode, nq, nk, h, d, offs, r.starts};

  hipError_t e;
  record(r, LT_STAGE_SAMPLE, st);
  if ((e = launch_init(qctl, st)) != hipSuccess) return hip_status(e);
  if ((e = make_list(r, nk, 1, list, st)) != hipSuccess) return hip_status(e);
  if (r.ns > 0 && (e = launch_sample_scores(a, list, r.ns, samp, st)) != hipSuccess) return hip_status(e);
  record(r, LT_STAGE_RANGE, st);
  if ((e = launch_range(false, samp, r.ns, nq, nk, offs, r.starts, list, r.ns, r.m, k, params, r.stats, rflag,
                        st)) != hipSuccess)
    return hip_status(e);
  record(r, LT_STAGE_FILTER, st);
  e = r.shared ? launch_wide_fused(a, params, r.S, r.L, r.cap, r.m, k, gate, cnt, hist, cand, st)
               : launch_fused_scan(a, params, r.S, r.L, r.cap, r.m, k, gate, cnt, hist, cand, nullptr, nullptr, st);
  if (e != hipSuccess) return hip_status(e);
  record(r, LT_STAGE_SELECT, st);
  // lists in arrival order: ties by key, every row sorted (also the rows the
  // fallback completes). Overflowed rows of the one-list-per-split scans get
  // a second filter pass at their final bin before any dense fallback.
  const bool refilter = !r.shared;
  const uint32_t sel_flags = r.flags | (sh.arrival_order ? kSelKeyed : 0u) | (r.shared ? kSelIlv : 0u) |
                             (refilter ? kSelRefilter : 0u);
  const uint32_t fb_flags = r.flags | (sh.arrival_order ? LT_SORTED_OUTPUT : 0u);
  if ((e = launch_select(params, cnt, hist, cand, nq, r.S, r.HS, r.cap, r.m, k, r.E, sel_flags, out_idx, out_scores,
                         qctl, queue, rqueue, rflag, r.stats, st)) != hipSuccess)
    return hip_status(e);
  record(r, LT_STAGE_FALLBACK, st);
  if (refilter) {
    if ((e = launch_fused_scan(a, params, r.S, r.L, r.cap, r.m, k, gate, cnt, hist, cand, rflag, qctl, st)) !=
        hipSuccess)
      return hip_status(e);
    if ((e = launch_select_second(params, cnt, hist, cand, nq, r.S, r.HS, r.cap, r.m, k, r.E, sel_flags, out_idx,
                                  out_scores, qctl, queue, rqueue, rflag, r.stats, st)) != hipSuccess)
      return hip_status(e);
  }
  const FallbackShape fs = fallback_shape(nq, nk);
  if ((e = launch_fused_fallback(a, k, fb_flags, qctl, queue, rflag + nq, fs.batch, fs.grid * fs.batch, scratch,
                                 fbc_idx, fbc_score, out_idx, out_scores, st)) != hipSuccess)
    return hip_status(e);
  // the dense fallback mode's selection (the wide scan's fallback has no
  // dense mode)
  if (!r.shared && (e = launch_fallback_rows(qctl, rflag + nq, scratch, nq, nk, offs, r.starts, k, fb_flags,
                                             fs.grid * fs.batch, sh.queries_per_block, out_idx, out_scores, st)) !=
                       hipSuccess)
    return hip_status(e);
  record(r, LT_NUM_STAGE_EVENTS - 1, st);
  return LT_OK;
}

int lt_indexer_topk_static(const void* q, const float* q_scale, const float* w, const void* keys,
                           const float* k_scale, lt_dtype dtype, lt_score_mode mode, int32_t nq, int32_t nk,
                           int32_t h, int32_t d, int32_t k, const int32_t* offs, int32_t* out_idx,
                           float* out_scores, const lt_options* opts, void* stream) {
  int rc = check_score_args(q, q_scale, keys, k_scale, dtype, mode, nq, nk, h, d);
  if (rc) return rc;
  if (k < 1) return LT_EINVAL;
  if (k > LT_K_MAX) return LT_EUNSUPPORTED;
  if (nq == 0) return LT_OK;
  const size_t need = lt_indexer_topk_workspace_size(nq, nk, h, d, dtype, mode, k, opts);
  if (need == 0) return LT_EINVAL;
  if (need > (size_t)LT_STATIC_SCRATCH_BYTES) return LT_ESCRATCH;
  void* ws = nullptr;
  if ((rc = static_scratch(&ws)) != LT_OK) return rc;
  return lt_indexer_topk(q, q_scale, w, keys, k_scale, dtype, mode, nq, nk, h, d, k, offs, out_idx, out_scores, ws,
                         (size_t)LT_STATIC_SCRATCH_BYTES, opts, stream);
}

int lt_indexer_scores(const void* q, const float* q_scale, const float* w, const void* keys,
                      const float* k_scale, lt_dtype dtype, lt_score_mode mode, int32_t nq, int32_t nk,
                      int32_t h, int32_t d, float* scores, int64_t ld, void* stream) {
  int rc = check_score_args(q, q_scale, keys, k_scale, dtype, mode, nq, nk, h, d);
  if (rc) return rc;
  if (ld < nk) return LT_EINVAL;
  if (nq == 0 || nk == 0) return LT_OK;
  if (!scores) return LT_EINVAL;
  ScoreArgs a{q, q_scale, w, keys, k_scale, (int)dtype, (int)mode, nq, nk, h, d, nullptr, nullptr};
  return hip_status(launch_dense_scores(a, scores, ld, (hipStream_t)stream));
}

size_t lt_topk_select_workspace_size(int32_t nq, int32_t nk, int32_t k, const lt_options* opts) {
  if (nq < 0 || nk < 0 || k < 1 || k > LT_K_MAX) return 0;
  Resolved r = resolve_scores(opts, nq, nk, k);
  if (r.status) return 0;
  return carve(nq, nk, r, false).total;
}

static int check_select_args(const float* scores, int64_t stride, int nq, int nk, int k) {
  if (nq < 0 || nk < 0 || k < 1) return LT_EINVAL;
  if (k > LT_K_MAX) return LT_EUNSUPPORTED;
  if (stride < nk || stride % 4 != 0) return LT_EINVAL;
  if (nq > 0 && nk > 0 && (!scores || !aligned(scores, 16))) return LT_EINVAL;
  return LT_OK;
}

int lt_topk_select(const float* scores, int64_t stride, int32_t nq, int32_t nk, int32_t k,
                   const int32_t* offs, int32_t* out_idx, float* out_scores, void* workspace,
                   size_t workspace_bytes, const lt_options* opts, void* stream) {
  int rc = check_select_args(scores, stride, nq, nk, k);
  if (rc) return rc;
  if (nq == 0) return LT_OK;
  if (!out_idx || !out_scores || !workspace || !aligned(workspace, 256)) return LT_EINVAL;
  const Resolved r = resolve_scores(opts, nq, nk, k);
  if (r.status) return r.status;
  const Layout L = carve(nq, nk, r, false);
  if (workspace_bytes < L.total) return LT_EWORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  uint32_t* qctl = reinterpret_cast<uint32_t*>(ws + L.qctl);
  int32_t* queue = reinterpret_cast<int32_t*>(ws + L.queue);
  RowParam* params = reinterpret_cast<RowParam*>(ws + L.params);
  int32_t* list = reinterpret_cast<int32_t*>(ws + L.list);
  uint32_t* cnt = reinterpret_cast<uint32_t*>(ws + L.cnt);
  uint32_t* hist = reinterpret_cast<uint32_t*>(ws + L.hist);
  int2* cand = reinterpret_cast<int2*>(ws + L.cand);
  int32_t* fbc_idx = reinterpret_cast<int32_t*>(ws + L.fbcand);
  float* fbc_score = reinterpret_cast<float*>(ws + L.fbcand + (size_t)kFallbackGrid * k * 4);

  hipError_t e;
  record(r, LT_STAGE_SAMPLE, st);
  if ((e = launch_init(qctl, st)) != hipSuccess) return hip_status(e);
  if ((e = make_list(r, nk, kSampleBlockScores, list, st)) != hipSuccess) return hip_status(e);
  record(r, LT_STAGE_RANGE, st);
  if ((e = launch_range(true, scores, stride, nq, nk, offs, r.starts, list, r.ns, r.m, k, params, r.stats, nullptr,
                        st)) != hipSuccess)
    return hip_status(e);
  record(r, LT_STAGE_FILTER, st);
  if ((e = launch_filter(scores, stride, nq, nk, offs, r.starts, params, r.S, r.L, r.cap, r.m, k, cnt, hist, cand,
                         st)) != hipSuccess)
    return hip_status(e);
  record(r, LT_STAGE_SELECT, st);
  if ((e = launch_select(params, cnt, hist, cand, nq, r.S, r.HS, r.cap, r.m, k, r.E, r.flags, out_idx, out_scores, qctl,
                         queue, nullptr, nullptr, r.stats, st)) != hipSuccess)
    return hip_status(e);
  record(r, LT_STAGE_FALLBACK, st);
  if ((e = launch_fallback_scores(scores, stride, nk, offs, r.starts, k, r.flags, qctl, queue, fbc_idx, fbc_score,
                                  out_idx, out_scores,
                                  std::min(std::max(nq, kFallbackGridScoresMin), kFallbackGridScoresMax), st)) !=
      hipSuccess)
    return hip_status(e);
  record(r, LT_NUM_STAGE_EVENTS - 1, st);
  return LT_OK;
}

int lt_topk_radix(const float* scores, int64_t stride, int32_t nq, int32_t nk, int32_t k,
                  const int32_t* offs, int32_t* out_idx, float* out_scores, uint32_t flags, void* stream) {
  int rc = check_select_args(scores, stride, nq, nk, k);
  if (rc) return rc;
  if (nq == 0) return LT_OK;
  if (!out_idx || !out_scores) return LT_EINVAL;
  return hip_status(launch_radix(scores, stride, nq, nk, offs, k, flags, out_idx, out_scores, (hipStream_t)stream));
}

size_t lt_sample_from_topk_workspace_size(int32_t nk) {
  if (nk < 0) return 0;
  return freq_workspace_bytes(nk);
}

int lt_sample_from_topk(const int32_t* prev, int64_t ld, int32_t rows, int32_t pk, int32_t nk, int32_t ns,
                        int32_t* out, void* workspace, size_t workspace_bytes, void* stream) {
  if (rows < 0 || pk < 0 || nk < 0 || ld < pk) return LT_EINVAL;
  if (ns < 1 || ns > LT_SAMPLE_LIST_MAX || !out) return LT_EINVAL;
  if ((int64_t)rows * pk >= (1LL << 31)) return LT_EINVAL;
  if (rows > 0 && pk > 0 && !prev) return LT_EINVAL;
  if (!workspace || !aligned(workspace, 256)) return LT_EINVAL;
  if (workspace_bytes < freq_workspace_bytes(nk)) return LT_EWORKSPACE;
  if (pk == 0) rows = 0;
  return hip_status(launch_sample_from_topk(prev, ld, rows, pk, nk, ns, out, workspace, (hipStream_t)stream));
}

int lt_dsa_union(const int32_t* idx, int64_t ld, int32_t nq, int32_t k, int32_t group, int32_t* union_idx,
                 int32_t* union_count, uint32_t* member_mask, void* stream) {
  if (nq < 0 || k < 1 || group < 1 || ld < k) return LT_EINVAL;
  if ((int64_t)group * k > LT_UNION_MAX) return LT_EINVAL;
  if (nq == 0) return LT_OK;
  if (!idx || !union_idx || !union_count || !member_mask) return LT_EINVAL;
  return hip_status(launch_dsa_union(idx, ld, nq, k, group, union_idx, union_count, member_mask,
                                     (hipStream_t)stream));
}

int lt_event_create(void** ev) {
  if (!ev) return LT_EINVAL;
  // timing only: no system-scope fence when the event completes, so that
  // recording one between two kernels does not write back and invalidate
  // the caches in between (which would show up as a gap in the timing)
  hipEvent_t e;
  if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return LT_EHIP;
  *ev = (void*)e;
  return LT_OK;
}

int lt_event_destroy(void* ev) { return hip_status(hipEventDestroy((hipEvent_t)ev)); }

int lt_event_record(void* ev, void* stream) { return hip_status(hipEventRecord((hipEvent_t)ev, (hipStream_t)stream)); }

int lt_event_elapsed_ms(void* a, void* b, float* ms) {
  if (!ms) return LT_EINVAL;
  if (hipEventSynchronize((hipEvent_t)b) != hipSuccess) return LT_EHIP;
  return hip_status(hipEventElapsedTime(ms, (hipEvent_t)a, (hipEvent_t)b));
}

}  // extern "C"
