/*
 * litetopk.h -- C ABI of the MI355X (gfx950) fused Indexer-TopK library.
 *
 * The library scores every causally visible key for every query with the DSA
 * indexer score and returns the exact per-row top-k, following the paper's
 * sample -> filter (bin, gate, online threshold refresh, batched write-back)
 * -> select workflow (sec. 3.1 "Overview", sec. 3.2), with an exact fallback
 * for rows whose candidate buffer overflows.
 *
 * Conventions shared by every entry point
 *  - Every array argument is a DEVICE pointer owned by the caller. The library
 *    never allocates or frees device memory, never synchronises the device or
 *    the stream, and keeps no state between calls: all scratch lives in the
 *    caller's workspace. Calls on different streams with different
 *    workspaces may run concurrently.
 *  - `stream` is a hipStream_t passed as an opaque pointer (NULL = the null
 *    stream). All work is enqueued on it in order; the call returns before the
 *    work finishes.
 *  - Argument checks happen on the host before anything is enqueued; a
 *    failing check returns a negative status and enqueues nothing. Device-side
 *    data problems (NaN or infinite scores) are not errors: they follow the
 *    total order below.
 *  - Total order used for selection (Eq. 2 of sec. 3.1 leaves ties open):
 *    higher score first; -0.0 equals +0.0; NaN ranks below -inf; equal scores
 *    go to the lower key index. The selected SET is therefore unique.
 *  - Output rows: row t holds min(k, e_t - s_t) selected entries followed by
 *    padding (index -1, score -inf). e_t = clamp(causal_offsets[t], 0,
 *    num_keys), or num_keys when causal_offsets is NULL; s_t = 0 unless
 *    lt_options.visible_start is set: row t sees keys [s_t, e_t). Scores are
 *    the raw float32 index scores I (never bin-space values). Without
 *    LT_SORTED_OUTPUT the selected entries come in an unspecified but
 *    deterministic order (the paper's select writes the above-threshold bins
 *    directly, sec. 3.2 "Top-k Selection"); with it they are sorted by the
 *    total order. Shapes with at most four heads (the one-head retrieval and
 *    768-dimensional shapes, the four-head float32 and bf16 shapes) always
 *    return sorted rows (their candidate lists fill in arrival order, so
 *    equal scores are told apart by the key itself), and report a zero score
 *    as +0.0 and a NaN score as the canonical quiet NaN.
 */
#ifndef LITETOPK_H
#define LITETOPK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
#define LT_OK 0
#define LT_EINVAL (-1)        /* bad pointer, size, stride, alignment or option   */
#define LT_EUNSUPPORTED (-2)  /* (dtype, heads, head_dim) not built, or k > LT_K_MAX */
#define LT_EWORKSPACE (-3)    /* workspace smaller than the *_workspace_size value */
#define LT_EHIP (-4)          /* a HIP launch or event call failed                 */
#define LT_ESCRATCH (-5)      /* lt_indexer_topk_static: the shape needs more workspace
                                 than LT_STATIC_SCRATCH_BYTES                      */

#define LT_K_MAX 8192         /* largest k (the paper's largest, sec. 4.1 retrieval) */
#define LT_MAX_BINS 256
#define LT_SAMPLE_LIST_MAX 32768  /* longest caller-supplied sample list */
#define LT_UNION_MAX 32768        /* largest group * k for lt_dsa_union */
#define LT_ROW_STATS 12           /* int32 fields per row of lt_options.row_stats */
#define LT_STATIC_SCRATCH_BYTES (256u << 20)  /* workspace of lt_indexer_topk_static, per GPU */

/* ---- enums --------------------------------------------------------------- */
typedef enum {
  LT_F32 = 0,         /* float32                                            */
  LT_BF16 = 1,        /* bfloat16                                           */
  LT_FP8_E4M3FN = 2   /* OCP FP8 E4M3FN bytes with per-token float32 scales */
} lt_dtype;

typedef enum {
  /* Eq. (1), sec. 2.1: I[t,s] = sum_j w[t,j] * ReLU(q[t,j] . k[s]) */
  LT_SCORE_DSA = 0,
  /* inner-product scorer (k-NN, sec. 3.1): I[t,s] = sum_j w[t,j] * (q[t,j] . k[s]) */
  LT_SCORE_IP = 1
} lt_score_mode;

/* flags for lt_options.flags */
#define LT_SORTED_OUTPUT 1u   /* sort every output row by the total order          */
#define LT_FORCE_FALLBACK 2u  /* send every row through the exact fallback path    */

/* Stage boundaries recorded into lt_options.stage_events when it is non-NULL:
   event i is recorded on `stream` before stage i, the last one after the last
   stage, so elapsed(event[i], event[i+1]) is the device time of stage i. */
#define LT_STAGE_SAMPLE 0     /* score / read the sample keys                  */
#define LT_STAGE_RANGE 1      /* per-row range, bin width and initial threshold */
#define LT_STAGE_FILTER 2     /* fused score + gate + write-back scan           */
#define LT_STAGE_SELECT 3     /* final selection from the candidate buffers     */
#define LT_STAGE_FALLBACK 4   /* exact fallback for overflowed rows             */
#define LT_NUM_STAGE_EVENTS 6

/* Tuning knobs. Pass NULL for the defaults; otherwise start from
   lt_options_default() and change fields. None of them changes a result. */
typedef struct lt_options {
  int32_t num_bins;        /* m, equal-width bins over the sample range (sec. 3.2
                              "Sampling"); 1..LT_MAX_BINS; default 256          */
  int32_t sample_size;     /* k': sampled keys per launch (sec. 3.2: k' = 3k for
                              DSA); negative = default: 3k in DSA mode,
                              max(3k, min(Nk/128, 65536)) in IP mode, max(3k,
                              65536) for the 768-dimensional IP shape (all
                              capped at Nk; the scores-in entry uses 3k); 0
                              disables the gate. With sample_keys set: the
                              length of that list, 1..LT_SAMPLE_LIST_MAX        */
  int32_t capacity;        /* candidate slots per (row, key split); <= 0 = default
                              max(12k, 2048) (sec. 4.2: 12k for k = 2048), and
                              k + max(1024, k/2) for the 768-dimensional shapes,
                              whose splits share one threshold (for those shapes
                              rounded up to a multiple of 16: their lists are
                              stored in chunks of 16 entries)                  */
  int32_t key_splits;      /* key-range splits per row; 0 = auto (fused), 1 (scores-in) */
  uint32_t flags;          /* LT_SORTED_OUTPUT | LT_FORCE_FALLBACK               */
  uint64_t seed;           /* seed of the key sample                             */
  void** stage_events;     /* NULL, or LT_NUM_STAGE_EVENTS hipEvent_t handles     */
  int32_t* row_stats;      /* NULL, or a DEVICE int32 [num_queries, LT_ROW_STATS]
                              receiving per row (the internal invariants of
                              sec. 3.2, for tests and tuning):
                              [0] candidates written (summed over splits);
                              [1] final threshold bin tau_f (-2 if the row was
                                  queued before it was found);
                              [2] how the row was completed: 0 by the
                                  final select; by the exact dense fallback
                                  because of 1 candidate buffer overflow,
                                  2 threshold bin too large to sort, 3 forced,
                                  4 candidate count disagrees with the
                                  histogram, 5 tau_f below the sample's
                                  initial bin (sample and scan scores
                                  disagree; sec. 3.2 "Sampling" guarantees
                                  tau_f >= tau0 otherwise); 6 buffer overflow
                                  finished by a second filter pass gated at
                                  the final bin tau_f (the histograms keep
                                  counting past the buffer, so tau_f is exact;
                                  shapes other than the 768-dimensional ones);
                              [3] candidates in bin tau_f;
                              [4] the sample's initial bin tau0 (-1 = no gate);
                              [5] bits of the float32 k-th largest visible
                                  sample score under the total order (-inf if
                                  fewer than k sample keys are visible);
                              [6], [7] bits of the float32 bin map (delta, c):
                                  a score I falls in bin
                                  floor(fmaf(I, delta, c)), clamped to
                                  m - 1 (below 0: not counted);
                              [8] m, the bins in use (num_bins, lowered where
                                  the shape's histograms would not fit in LDS);
                              [9] sample keys visible to the row;
                              [10], [11] 0.
                              Fields 4-11 are written for every row, 0-3 by
                              the final select or when the row is queued.
                              Collecting them adds passes over the sample.  */
  const int32_t* sample_keys; /* NULL = a random stratified sample drawn with
                              `seed`; else a DEVICE int32 [sample_size] list of
                              key indices to score as the sample instead. Sec. 3.2
                              "Sampling" reuses the keys that occur most often in
                              the previous chunk's top-k (lt_sample_from_topk).
                              Any list gives exact results: entries outside
                              [0, num_keys) and repeated entries are dropped, and
                              row t uses only the entries below e_t. The list is
                              read on the stream; it must stay valid until the
                              call's work has run.                              */
  const int32_t* visible_start; /* NULL, or a DEVICE int32 [num_queries]: row t
                              sees keys [s_t, e_t) with s_t =
                              clamp(visible_start[t], 0, e_t) -- several
                              sequences packed into one key array, each query
                              seeing its own sequence. NULL = 0.                */
} lt_options;

/* Fills *opts with the defaults (k-dependent fields are resolved per call). */
void lt_options_default(lt_options* opts);

/* ---- fused Indexer-TopK ------------------------------------------------- */

/* Bytes of device workspace lt_indexer_topk needs for this shape. Returns 0
   for an invalid or unsupported shape. */
size_t lt_indexer_topk_workspace_size(int32_t num_queries, int32_t num_keys, int32_t num_heads,
                                      int32_t head_dim, lt_dtype dtype, lt_score_mode mode,
                                      int32_t k, const lt_options* opts);

/* Exact per-row top-k of the index score (Eq. 1 for LT_SCORE_DSA, the inner
   product for LT_SCORE_IP) over the visible keys, Eq. (2), computed by the
   fused sample / filter / select pipeline of sec. 3.2 without materialising
   the score matrix.

   q         [num_queries, num_heads, head_dim] in `dtype`, row-major (for fp8:
             E4M3FN bytes). 16-byte aligned.
   q_scale   [num_queries, num_heads] float32 > 0, fp8 only (NULL otherwise).
   w         [num_queries, num_heads] float32 head weights w[t,j]; NULL = all 1.
   keys      [num_keys, head_dim] in `dtype`, row-major. 16-byte aligned.
   k_scale   [num_keys] float32 > 0, fp8 only (NULL otherwise).
             For fp8 the scales multiply the decoded values; they must be
             positive so that they factor out of the ReLU.
   k         1..LT_K_MAX.
   causal_offsets  [num_queries] int32 or NULL (see the row convention above).
   out_idx   [num_queries, k] int32;  out_scores [num_queries, k] float32.
   workspace at least lt_indexer_topk_workspace_size(...) bytes, 256-byte aligned;
             its contents on entry do not matter.
   Supported (dtype, mode, num_heads, head_dim): f32 DSA (4, 64), f32 DSA and IP
   (1, 64); bf16 DSA (64, 128), bf16 DSA (4, 128), bf16 DSA and IP (1, 128);
   bf16 DSA and IP (1, 768) (the retrieval shapes of sec. 4.1); fp8 DSA
   (64, 128). Anything else returns LT_EUNSUPPORTED. */
int lt_indexer_topk(const void* q, const float* q_scale, const float* w, const void* keys,
                    const float* k_scale, lt_dtype dtype, lt_score_mode mode, int32_t num_queries,
                    int32_t num_keys, int32_t num_heads, int32_t head_dim, int32_t k,
                    const int32_t* causal_offsets, int32_t* out_idx, float* out_scores,
                    void* workspace, size_t workspace_bytes, const lt_options* opts, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
   capture, tight serving loops, harnesses that forbid hipMalloc): the same
   operation, arguments and results as lt_indexer_topk, with the workspace
   taken from a static device array of LT_STATIC_SCRATCH_BYTES that the library
   holds on every GPU it runs on until the process ends. The call allocates
   nothing. It uses the array of the device current on the calling thread
   (the stream must belong to that device); its address is looked up on the
   first call made on each device.
   Returns LT_ESCRATCH, before any device work, when
   lt_indexer_topk_workspace_size(...) of the shape exceeds
   LT_STATIC_SCRATCH_BYTES, and the argument errors of lt_indexer_topk.
   Every call on one GPU shares that GPU's array: calls whose work overlaps
   (on different streams, or from different threads without ordering) race
   and give undefined results. Calls ordered on one stream are safe; each
   call initialises what it reads from the array. */
int lt_indexer_topk_static(const void* q, const float* q_scale, const float* w, const void* keys,
                           const float* k_scale, lt_dtype dtype, lt_score_mode mode, int32_t num_queries,
                           int32_t num_keys, int32_t num_heads, int32_t head_dim, int32_t k,
                           const int32_t* causal_offsets, int32_t* out_idx, float* out_scores,
                           const lt_options* opts, void* stream);

/* ---- dense scores (the decoupled baseline's score stage, sec. 1) --------- */

/* Writes the float32 index score of every (query, key) pair, visible or not,
   to scores[t * ld + s] for s < num_keys (ld >= num_keys). Same arguments and
   supported shapes as lt_indexer_topk; the arithmetic is bit-identical to the
   fused scan's, so lt_topk_select over this matrix returns exactly what
   lt_indexer_topk returns. This is the materialising path the paper's
   method exists to avoid; it serves as the unfused baseline and for tests. */
int lt_indexer_scores(const void* q, const float* q_scale, const float* w, const void* keys,
                      const float* k_scale, lt_dtype dtype, lt_score_mode mode,
                      int32_t num_queries, int32_t num_keys, int32_t num_heads, int32_t head_dim,
                      float* scores, int64_t ld, void* stream);

/* ---- scores-in selection --------------------------------------------------- */

size_t lt_topk_select_workspace_size(int32_t num_queries, int32_t num_keys, int32_t k,
                                     const lt_options* opts);

/* Exact per-row top-k (Eq. 2) of a float32 score matrix: scores[t * row_stride
   + s], s < num_keys (row_stride >= num_keys, 16-byte aligned rows, i.e.
   row_stride % 4 == 0). Uses the same sample / bin / gate / refresh / select
   pipeline as the fused entry, streaming the scores from HBM once. Bit-exact:
   the output entries are input values, chosen under the total order. */
int lt_topk_select(const float* scores, int64_t row_stride, int32_t num_queries, int32_t num_keys,
                   int32_t k, const int32_t* causal_offsets, int32_t* out_idx, float* out_scores,
                   void* workspace, size_t workspace_bytes, const lt_options* opts, void* stream);

/* Exact per-row top-k of a float32 score matrix by plain radix selection over
   all visible scores, with no sampling or filtering (the decoupled designs'
   selector, sec. 1 and sec. 3.2 "Top-k Selection"). Needs no workspace.
   `flags` accepts LT_SORTED_OUTPUT. Same layout rules as lt_topk_select. */
int lt_topk_radix(const float* scores, int64_t row_stride, int32_t num_queries, int32_t num_keys,
                  int32_t k, const int32_t* causal_offsets, int32_t* out_idx, float* out_scores,
                  uint32_t flags, void* stream);

/* ---- sample from the previous chunk (sec. 3.2 "Sampling") ---------------- */

/* Bytes of device workspace lt_sample_from_topk needs for num_keys keys
   (0 for num_keys < 0). */
size_t lt_sample_from_topk_workspace_size(int32_t num_keys);

/* The sample the paper takes for a prefill chunk: the keys that occur most
   often in the previous chunk's top-k results. count(s) is the number of
   entries prev_idx[t * ld + j] == s over t < prev_rows, j < prev_k; entries
   outside [0, num_keys) (such as the -1 padding) are ignored. The selected
   keys are the sample_size keys of largest count (equal counts: lower key
   index first), restricted to keys with count >= 1. They are written to
   sample_keys[0, n) in ascending key order, followed by -1 up to
   sample_size. The result is meant as lt_options.sample_keys for the next
   chunk of queries over the same keys (any list is safe there).
   prev_idx    DEVICE int32, rows of `ld` >= prev_k entries (prev_rows may be 0).
   sample_keys DEVICE int32 [sample_size]; 1 <= sample_size <= LT_SAMPLE_LIST_MAX.
   workspace   at least lt_sample_from_topk_workspace_size(num_keys) bytes,
               256-byte aligned; contents on entry do not matter.
   Limits: prev_rows * prev_k < 2^31. */
int lt_sample_from_topk(const int32_t* prev_idx, int64_t ld, int32_t prev_rows, int32_t prev_k,
                        int32_t num_keys, int32_t sample_size, int32_t* sample_keys, void* workspace,
                        size_t workspace_bytes, void* stream);

/* ---- LiteDSA union and membership masks (sec. 3.3) ------------------------ */

/* For each group of `group` consecutive queries (the last group may be
   shorter), the union of their top-k key lists as one ascending list of
   distinct keys shared by the group, and for every query a bitmask over the
   union's slots marking the keys of its own top-k (the per-query membership
   mask LiteDSA's attention ANDs with each row, sec. 3.3).
   topk_idx     DEVICE int32, query t's list at topk_idx[t * ld + j], j < k
                (ld >= k); negative entries (the -1 padding) are not keys;
                repeated keys in one list count once.
   union_idx    DEVICE int32 [ceil(num_queries / group), group * k]: row g
                holds group g's union ascending, then -1.
   union_count  DEVICE int32 [ceil(num_queries / group)]: union sizes.
   member_mask  DEVICE uint32 [num_queries, W], W = ceil(group * k / 32):
                bit (j % 32) of word j / 32 of row t is set iff union slot j
                of t's group holds a key of t's list; bits past the union
                size are 0.
   Limits: 1 <= group, 1 <= k, group * k <= LT_UNION_MAX. No workspace. */
int lt_dsa_union(const int32_t* topk_idx, int64_t ld, int32_t num_queries, int32_t k, int32_t group,
                 int32_t* union_idx, int32_t* union_count, uint32_t* member_mask, void* stream);

/* ---- timing helpers ------------------------------------------------------- */

/* Thin wrappers over hipEventCreateWithFlags / hipEventDestroy /
   hipEventElapsedTime / hipEventRecord / hipEventSynchronize for callers
   without a HIP binding. The events are for timing only: they are created
   with hipEventDisableSystemFence, so recording one between two kernels adds
   no cache write-back, and waiting on one does not make device writes
   visible to the host (synchronise the stream for that). */
int lt_event_create(void** event);
int lt_event_destroy(void* event);
int lt_event_record(void* event, void* stream);
int lt_event_elapsed_ms(void* start, void* stop, float* ms);  /* synchronises on stop */

/* Human-readable text for a status code. */
const char* lt_strerror(int status);

#ifdef __cplusplus
}
#endif
#endif /* LITETOPK_H */
