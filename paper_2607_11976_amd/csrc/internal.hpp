// Internal interface between the C ABI (abi.hip) and the kernel translation
// units. Not installed; the public interface is include/litetopk.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/litetopk.h"
#include "common.hpp"

namespace lt {

// ---- selection side (select.hip) ----
hipError_t launch_init(uint32_t* qctl, hipStream_t st);
// Visibility: row t sees keys [s_t, e_t) (row_range); `offs` holds the ends
// (NULL = num_keys) and `starts` the starts (NULL = 0).
// With stats non-NULL, also writes row_stats fields 4..11 (the sample's
// initial bin and k-th score, the bin map, the bins in use).
// rflag (or NULL): [2 * nq] per-row flags, cleared here: [0, nq) the second
// filter pass, [nq, 2 nq) the dense fallback (set by the select when it
// queues a row there).
hipError_t launch_range(bool from_scores, const float* src, int64_t stride, int nq, int nk,
                        const int32_t* offs, const int32_t* starts, const int32_t* list, int ns, int m, int k,
                        RowParam* params, int32_t* stats, int32_t* rflag, hipStream_t st);
hipError_t launch_filter(const float* scores, int64_t stride, int nq, int nk, const int32_t* offs,
                         const int32_t* starts, const RowParam* params, int S, int L, int cap, int m, int k,
                         uint32_t* cnt, uint32_t* hist, int2* cand, hipStream_t st);
size_t select_lds_bytes(int E);
// S candidate lists per row (cnt [nq, S], cand [nq, S, cap]); HS histograms
// per row (hist [nq, HS, m]), HS = S or 1.
// Rows that need the dense fallback go to queue (count qctl[0]); with
// kSelRefilter in flags, overflowed rows whose final bins fit go to rqueue
// (count qctl[1]) with rflag set and params[row].tau0 = their final bin.
hipError_t launch_select(RowParam* params, const uint32_t* cnt, const uint32_t* hist, const int2* cand, int nq,
                         int S, int HS, int cap, int m, int k, int E, uint32_t flags, int32_t* out_i, float* out_s,
                         uint32_t* qctl, int32_t* queue, int32_t* rqueue, int32_t* rflag, int32_t* stats,
                         hipStream_t st);
// The select of the rows in rqueue after their second filter pass.
hipError_t launch_select_second(RowParam* params, const uint32_t* cnt, const uint32_t* hist, const int2* cand,
                                int nq, int S, int HS, int cap, int m, int k, int E, uint32_t flags, int32_t* out_i,
                                float* out_s, uint32_t* qctl, int32_t* queue, int32_t* rqueue, int32_t* rflag,
                                int32_t* stats, hipStream_t st);
// Exact fallback of the scores-in entry for the queued rows (queue, length
// qctl[0]), radix selection straight from the caller's score rows, `grid`
// blocks: few rows (fallback_chunks over min(grid, kFallbackGrid) blocks)
// have their visible keys cut into chunks, one block per (row, chunk), each
// selecting its chunk's top-k into cidx / cscore [kFallbackGrid * k] and
// counting the chunk on qctl[kQctlDone + entry], the last one selecting the
// row from the chunks' candidates; otherwise one block per row.
hipError_t launch_fallback_scores(const float* scores, int64_t stride, int nk, const int32_t* offs,
                                  const int32_t* starts, int k, uint32_t flags, uint32_t* qctl,
                                  const int32_t* queue, int32_t* cidx, float* cscore, int32_t* out_i, float* out_s,
                                  int grid, hipStream_t st);
hipError_t launch_radix(const float* scores, int64_t stride, int nq, int nk, const int32_t* offs,
                        int k, uint32_t flags, int32_t* out_i, float* out_s, hipStream_t st);

// ---- sample lists (sample.hip) ----
// list[i] = the i-th key of the stratified random sample (runs of blk keys).
hipError_t launch_sample_list(int32_t* list, int ns, int nk, int blk, uint64_t seed, hipStream_t st);
// out = the caller's list with out-of-range and repeated keys replaced by -1 (ns <= LT_SAMPLE_LIST_MAX).
hipError_t launch_list_clean(const int32_t* in, int ns, int nk, int32_t* out, hipStream_t st);
// The previous-chunk sample (lt_sample_from_topk); ws holds freq_workspace_bytes(nk).
size_t freq_workspace_bytes(int nk);
hipError_t launch_sample_from_topk(const int32_t* prev, int64_t ld, int rows, int pk, int nk, int ns,
                                   int32_t* out, void* ws, hipStream_t st);

// ---- LiteDSA union (union.hip) ----
size_t union_lds_bytes(int group, int k);
hipError_t launch_dsa_union(const int32_t* idx, int64_t ld, int nq, int k, int group, int32_t* uidx, int32_t* ucount,
                            uint32_t* mask, hipStream_t st);

// ---- score side (score.hip) ----
struct ScoreArgs {
  const void* q;
  const float* q_scale;
  const float* w;
  const void* keys;
  const float* k_scale;
  int dtype, mode, nq, nk, h, d;
  const int32_t* offs;    // row ends (NULL = nk)
  const int32_t* starts;  // row starts (NULL = 0)
};

// Static shape of one compiled score configuration.
struct ScoreShape {
  int supported;
  int queries_per_block;  // queries one block owns
  int keys_per_step;      // keys per LDS tile
  int threads;            // block size
  size_t scan_lds;        // LDS bytes of the fused scan (tiles, per-query state), excluding histograms
  int shared_rows;        // 1: all key splits of a row share one histogram,
                          // threshold and candidate list (the wide scan)
  int arrival_order;      // 1: candidate lists fill in arrival order, not key
                          // order (the grouped and wide scans)
};
ScoreShape score_shape(int dtype, int mode, int h, int d);

// Sample scores: samp[t * ns + i] = I(t, list[i]) (holes score key 0; never read).
hipError_t launch_sample_scores(const ScoreArgs& a, const int32_t* list, int ns, float* samp, hipStream_t st);
// Dense scores: out[t * ld + s] = I(t, s) for every key.
hipError_t launch_dense_scores(const ScoreArgs& a, float* out, int64_t ld, hipStream_t st);
// Fused score + gate + write-back scan over S key splits of L keys each;
// pub [nq * 8 bytes] holds the bins the splits of each row publish where they
// share thresholds (initialised here).
// rflag NULL: every row. Else the second filter pass: only rows with
// rflag[t] set are scanned and written (blocks without such rows, and every
// block when qctl[1] == 0, return at once).
hipError_t launch_fused_scan(const ScoreArgs& a, const RowParam* params, int S, int L, int cap, int m,
                             int k, int* pub, uint32_t* cnt, uint32_t* hist, int2* cand, const int32_t* rflag,
                             const uint32_t* qctl, hipStream_t st);
// Exact fallback for queued rows (queue, length qctl[0]): dense re-score
// into scratch rows of nk floats (`slots` of them), then radix select. The
// fallback kernel runs kFallbackGrid blocks in one of three modes (the wide
// scan's, in the split or whole-row mode), chosen on the device from the
// queue length n:
// * split (fallback_chunks(...) > 1: few rows, each with its own scratch
//   row): the visible keys of every queued row are cut into that many chunks,
//   one block per (row, chunk), which also selects its chunk's top-k into
//   the candidate arrays; the block that completes a row's last chunk
//   (counter qctl[kQctlDone + entry]) selects the row from its chunks'
//   candidates.
// * dense (fallback_dense(...): every row of the call has a scratch row of
//   its own, nq <= slots): the blocks take (query tile, key slice) items of
//   the tiles holding queued rows, slice by slice, and write each queued row
//   t's scores to scratch row t, every tile scored once; launch_fallback_rows
//   then radix-selects each queued row, one block per row.
// * whole rows: blocks below slots / batch take queue entries from the
//   cursor qctl[kQctlCursor] and re-score whole rows into their own scratch
//   rows [blockIdx][batch][nk]. fbflag (or NULL) [nq]: 1 for the queued rows;
//   a block that takes a row also claims up to batch - 1 other queued rows of
//   the same query tile (1 -> 2) and re-scores them in the same pass.
// qctl words: [0] fallback queue length, [1] second-pass queue length,
// [kQctlCursor] the whole-row cursor, [kQctlDone, + kMaxSplitRows) the split
// mode's chunk counters; all zeroed by launch_init.
constexpr int kMaxFallbackBatch = 8;  // rows of one query tile re-scored in one fallback pass
constexpr int kFallbackGrid = 256;    // blocks of a fallback launch
constexpr int kQctlWords = 256;
constexpr int kQctlCursor = 2;
constexpr int kQctlDone = 4;
constexpr int kMaxSplitRows = kFallbackGrid / 2;
constexpr int kSplitMinKeys = 4096;  // keys per chunk at least
static_assert(kQctlDone + kMaxSplitRows <= kQctlWords, "chunk counters must fit in qctl");
// Chunks per queued row in split mode, or 1 (whole-row mode): split when at
// least two blocks per row are available, every row has a scratch row of its
// own, and the chunks keep kSplitMinKeys keys.
__host__ __device__ inline int fallback_chunks(uint32_t n, int grid, int slots, int nk) {
  if (n == 0 || n > (uint32_t)kMaxSplitRows || n > (uint32_t)slots || 2 * n > (uint32_t)grid) return 1;
  int c = grid / (int)n;
  const int by_keys = nk / kSplitMinKeys;
  if (c > by_keys) c = by_keys;
  return c < 2 ? 1 : c;
}
// Dense mode (see above): any queue the split mode does not take, when every
// row has a scratch row and the scan's query tiles hold at most 64 rows (the
// tile's row slots are bytes). kDenseSlice keys per item.
constexpr int kDenseSlice = 8192;
__host__ __device__ inline bool fallback_dense(uint32_t n, int nq, int grid, int slots, int nk, int qt) {
  return n > 0 && qt <= 64 && nq <= slots && fallback_chunks(n, grid, slots, nk) == 1;
}
// cidx / cscore [kFallbackGrid * k]: the split mode's chunk candidates.
hipError_t launch_fused_fallback(const ScoreArgs& a, int k, uint32_t flags, uint32_t* qctl, const int32_t* queue,
                                 int32_t* fbflag, int batch, int slots, float* scratch, int32_t* cidx, float* cscore,
                                 int32_t* out_i, float* out_s, hipStream_t st);
// The dense mode's selection: a block per row t < nq whose fallback flag
// fbflag[t] is 1 radix-selects scratch row t over the row's visible keys
// (offs / starts as in ScoreArgs) into out_i / out_s [nq][k]; every block
// returns at once unless fallback_dense(qctl[0], nq, kFallbackGrid, slots,
// nk, qt) holds. The host launches it only where that can hold.
hipError_t launch_fallback_rows(const uint32_t* qctl, const int32_t* fbflag, const float* scratch, int nq, int nk,
                                const int32_t* offs, const int32_t* starts, int k, uint32_t flags, int slots,
                                int qt, int32_t* out_i, float* out_s, hipStream_t st);

// ---- wide-vector scan (wide.hip): bf16, one head, long vectors ----
// wide_shape(...).supported is 0 for shapes the wide scan does not build.
ScoreShape wide_shape(int dtype, int mode, int h, int d);
hipError_t launch_wide_sample(const ScoreArgs& a, const int32_t* list, int ns, float* samp, hipStream_t st);
hipError_t launch_wide_dense(const ScoreArgs& a, float* out, int64_t ld, hipStream_t st);
// Fused scan with shared row state: gate [nq] (published threshold bins) and
// hist [nq, m] shared by the S key splits of a row (initialised here); cnt
// [nq, S] and cand [nq, S, cap] hold each split's own list, as in
// launch_fused_scan.
hipError_t launch_wide_fused(const ScoreArgs& a, const RowParam* params, int S, int L, int cap, int m, int k,
                             int* gate, uint32_t* cnt, uint32_t* hist, int2* cand, hipStream_t st);
hipError_t launch_wide_fallback(const ScoreArgs& a, int k, uint32_t flags, uint32_t* qctl, const int32_t* queue,
                                int slots, float* scratch, int32_t* cidx, float* cscore, int32_t* out_i, float* out_s,
                                hipStream_t st);

// k_select flags (internal).
// kSelKeyed: candidate lists are not in key order (the grouped and wide scans
// fill them in arrival order), so equal scores are ordered by the key itself,
// every row is output sorted and its scores are rebuilt from the sort keys.
// kSelIlv: the lists are stored interleaved in chunks of 16 (ilv_index, the
// wide scan); rows are few and long, so the select runs 1024-thread blocks.
constexpr uint32_t kSelKeyed = 1u << 30;
constexpr uint32_t kSelIlv = 1u << 29;
// kSelRefilter: a row whose lists overflowed but whose keys at or above its
// final bin fit in one list is queued for a second filter pass gated at that
// bin (rqueue, qctl[1], rflag) instead of the dense fallback.
// kSelSecond: the select of the rows of that second pass.
constexpr uint32_t kSelRefilter = 1u << 28;
constexpr uint32_t kSelSecond = 1u << 27;

}  // namespace lt
