// Device helpers shared by the LiteTopK kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lt {

constexpr int kWave = 64;
// Word 3 of a raw buffer descriptor on gfx950 (32-bit data, no swizzle, no
// stride): offsets are byte offsets range-checked against the record count.
constexpr int kBufferRaw = 0x00020000;
constexpr int kMaxBins = 256;

// Candidate lists of the shared-threshold (768-d) scan: `nlists` lists of
// `cap` entries (cap a multiple of 16) stored in 128-byte chunks of 16
// entries, chunk c of every list before chunk c + 1 of any. The lists grow
// a few entries at a time in every block, so the chunks being appended to sit
// together in a few megabytes instead of one page per list.
__host__ __device__ constexpr int64_t ilv_index(int64_t list, uint32_t pos, int64_t nlists) {
  return (int64_t)(pos >> 4) * nlists * 16 + list * 16 + (pos & 15u);
}

// ---------------------------------------------------------------------------
// Total order on float32 scores (selection, Eq. 2 with ties made unique):
// higher first, -0 == +0, NaN below -inf. ord_key maps a score to an unsigned
// key with the same order; NaN is the only value mapped to 0.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t ord_key(float f) {
  uint32_t b = __float_as_uint(f);
  if (f != f) return 0u;
  if (b == 0x80000000u) b = 0u;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Composite 64-bit key: larger = earlier in the output order. `pos` is any
// position that increases with the key index (ties go to the smaller pos).
__device__ __forceinline__ uint64_t comp_key(float score, uint32_t pos) {
  return ((uint64_t)ord_key(score) << 32) | (uint64_t)(0xFFFFFFFFu - pos);
}
__device__ __forceinline__ uint32_t comp_pos(uint64_t ck) { return 0xFFFFFFFFu - (uint32_t)ck; }

// ---------------------------------------------------------------------------
// Key sample (sec. 3.2 "Sampling": for workloads without temporal structure a
// random sample suffices). Sample slot i in [0, ns) maps to a distinct key:
// the ns slots form ceil(ns/blk) blocks of blk consecutive keys, block j is
// placed at a hashed offset inside the j-th equal stratum of [0, nk).
// Distinct because the strata are disjoint and each holds its whole block.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t mix32(uint64_t x) {
  x += 0x9E3779B97F4A7C15ull;
  x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
  x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
  x ^= x >> 31;
  return (uint32_t)(x >> 32);
}

// Number of sample slots actually used for nk keys and a requested size.
__host__ __device__ __forceinline__ int sample_count(int requested, int nk) {
  return requested < nk ? requested : nk;
}

__device__ __forceinline__ int sample_key(int i, int ns, int nk, int blk, uint64_t seed) {
  if (ns >= nk) return i;                       // the sample is every key
  int nb = (ns + blk - 1) / blk;                // blocks
  if ((int64_t)nb * blk > nk) {                 // strata too short for whole blocks:
    blk = 1;                                    // fall back to one key per stratum
    nb = ns;
  }
  int j = i / blk, o = i - j * blk;
  int len = (j == nb - 1) ? ns - j * blk : blk; // last block may be short
  int64_t lo = (int64_t)j * nk / nb, hi = (int64_t)(j + 1) * nk / nb;
  int64_t room = hi - lo - len + 1;             // >= 1: every stratum holds >= blk keys
  uint32_t r = mix32(seed * 0x632BE59BD9B4E019ull + (uint64_t)j);
  return (int)(lo + (int64_t)(r % (uint64_t)room)) + o;
}

// Visible key range [s, e) of a row: e = clamp(end[row], 0, nk) (nk without
// ends), s = clamp(start[row], 0, e) (0 without starts).
struct RowRange {
  int s, e;
};
__device__ __forceinline__ RowRange row_range(const int32_t* ends, const int32_t* starts, int row, int nk) {
  int e = ends ? ends[row] : nk;
  e = e < 0 ? 0 : (e > nk ? nk : e);
  int s = starts ? starts[row] : 0;
  s = s < 0 ? 0 : (s > e ? e : s);
  return RowRange{s, e};
}


// ---------------------------------------------------------------------------
// Equal-width bins (sec. 3.2 "Sampling"): bin = floor((I - s_min) * delta),
// evaluated as x = fma(I, delta, c) with c = -s_min * delta. Any such x is
// non-decreasing in I (delta > 0, rounding is monotone), which is all the
// exactness argument needs. Scores below the range (and NaN) get bin -1;
// scores above it are clamped into the top bin m-1.
// ---------------------------------------------------------------------------
struct RowParam {
  float delta;   // 1 / bin width (> 0, finite)
  float c;       // -s_min * delta (finite)
  int tau0;      // initial threshold bin from the sample, -1 = no gate
  int nsample;   // visible sample keys of the row
};

__device__ __forceinline__ float bin_x(float I, float delta, float c) { return fmaf(I, delta, c); }

__device__ __forceinline__ int bin_of(float x, int m) {
  if (!(x >= 0.0f)) return -1;
  if (x >= (float)(m - 1)) return m - 1;
  return (int)x;
}

// Gate threshold for bin tau: bin(x) >= tau  <=>  !(x < thr(tau)) for tau >= 0;
// tau = -1 lets everything through (NaN included).
__device__ __forceinline__ float gate_thr(int tau) {
  return tau >= 0 ? (float)tau : -__builtin_inff();
}

// ---------------------------------------------------------------------------
// Wave-level helpers
// ---------------------------------------------------------------------------
__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

__device__ __forceinline__ uint32_t mbcnt64(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ uint32_t wave_suffix_sum_excl(uint32_t v) {
  // sum of v over lanes strictly above this one
  const int l = lane_id();
  uint32_t s = v;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    uint32_t t = __shfl_down(s, off, kWave);
    if (l + off < kWave) s += t;
  }
  return s - v;
}

__device__ __forceinline__ float wave_min(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fminf(v, __shfl_xor(v, off, kWave));
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, kWave));
  return v;
}
__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

// OR of a 32-bit value over the wave: inclusive scans in rows of 16 lanes,
// then across rows (row_bcast); lane 63 ends with the total.
__device__ __forceinline__ uint32_t wave_or(uint32_t v) {
  v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false);  // row_shr:1
  v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false);  // row_shr:2
  v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false);  // row_shr:4
  v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false);  // row_shr:8
  v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);  // row_bcast:15
  v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// Inclusive prefix sum over the lanes of the wave: scans within rows of 16
// lanes (row_shr), then across rows (row_bcast), on the DPP path.
__device__ __forceinline__ uint32_t wave_prefix_sum(uint32_t v) {
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false);  // row_shr:1
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false);  // row_shr:2
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false);  // row_shr:4
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false);  // row_shr:8
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);  // row_bcast:15
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return v;
}

// Threshold refresh (sec. 3.2 "Threshold Refresh"): walk the histogram from
// the top bin down until the running count reaches k. Returns the largest bin
// b with sum_{b' >= b} hist[b'] >= k, or -1 if there is none, and the count of
// the bins strictly above it in *above. Called by a whole wave; lane l holds
// bins [4l, 4l + 4) in h[] (zero past the last bin).
__device__ __forceinline__ int wave_threshold_vals(const uint32_t (&h)[4], uint32_t k, uint32_t* above) {
  const uint32_t tot = h[0] + h[1] + h[2] + h[3];
  const uint32_t incl = wave_prefix_sum(tot);
  const uint32_t excl = (uint32_t)__builtin_amdgcn_readlane((int)incl, kWave - 1) - incl;  // lanes above this one
  uint32_t suf[4];
  suf[3] = excl + h[3];
  suf[2] = suf[3] + h[2];
  suf[1] = suf[2] + h[1];
  suf[0] = suf[1] + h[0];
  int nge = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) nge += __popcll(__ballot(suf[j] >= k));
  const int tau = nge - 1;
  if (above) {
    // count strictly above tau: the suffix of bin tau + 1 (0 past the end)
    const int want = tau + 1, j = want & 3;
    const uint32_t v = j == 0 ? suf[0] : j == 1 ? suf[1] : j == 2 ? suf[2] : suf[3];
    *above = want < 4 * kWave ? (uint32_t)__builtin_amdgcn_readlane((int)v, want >> 2) : 0u;
  }
  return tau;
}

// The same walk over a histogram of m bins in memory (LDS or global).
template <typename P>
__device__ __forceinline__ int wave_threshold(P hist, int m, uint32_t k, uint32_t* above) {
  const int l = lane_id();
  uint32_t h[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    int b = 4 * l + j;
    h[j] = b < m ? hist[b] : 0u;
  }
  return wave_threshold_vals(h, k, above);
}

// Inverse of ord_key on its image: the float with that order key (NaN maps
// back to the canonical quiet NaN, and -0 was already merged into +0).
__device__ __forceinline__ float ord_inv(uint32_t u) {
  if (u == 0u) return __builtin_nanf("");
  return __uint_as_float((u & 0x80000000u) ? (u & 0x7FFFFFFFu) : ~u);
}

}  // namespace lt
