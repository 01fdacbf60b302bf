// Block-level selection routines: ordered compaction, bitonic sort and exact
// radix selection of one row. Used by the final select, the fallback paths
// and the plain radix-select entry.
#pragma once

#include "common.hpp"

namespace lt {

// Exclusive prefix sum over the block in thread order; *total receives the
// block sum. `tmp` is LDS scratch of at least NTH/64 words. Contains two
// __syncthreads, so every thread of the block must call it.
template <int NTH>
__device__ __forceinline__ uint32_t block_scan_excl(uint32_t v, uint32_t* tmp, uint32_t* total) {
  constexpr int NW = NTH / kWave;
  const int l = lane_id(), w = threadIdx.x / kWave;
  uint32_t s = v;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    uint32_t t = __shfl_up(s, off, kWave);
    if (l >= off) s += t;
  }
  if (l == kWave - 1) tmp[w] = s;
  __syncthreads();
  uint32_t base = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    uint32_t x = tmp[i];
    if (i < w) base += x;
    tot += x;
  }
  __syncthreads();
  *total = tot;
  return base + s - v;
}

// Descending bitonic sort of P (power of two) unsigned keys in LDS.
template <int NTH, typename T>
__device__ __forceinline__ void bitonic_sort_desc(T* a, int P) {
  for (int size = 2; size <= P; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int t = threadIdx.x; t < (P >> 1); t += NTH) {
        int i = 2 * t - (t & (stride - 1));
        int j = i + stride;
        bool desc = (i & size) == 0;
        T x = a[i], y = a[j];
        if ((x < y) == desc) {
          a[i] = y;
          a[j] = x;
        }
      }
      __syncthreads();
    }
  }
}

__host__ __device__ __forceinline__ int next_pow2(int n) {
  int p = 1;
  while (p < n) p <<= 1;
  return p;
}

// LDS bytes radix_select_row needs for a given k.
__host__ __device__ __forceinline__ size_t radix_lds_bytes(int k) {
  return 256 * 4 + 64 + (size_t)next_pow2(k) * 8;
}

// Sort the first n (<= k) entries of an output row by the total order, in
// place. The rows were written by this block; the caller has made them
// visible with a block-scope fence and barrier. `fetch(idx)` returns the score
// of key idx (used to rebuild the float exactly, -0 and NaN payloads included).
template <int NTH, class Fetch>
__device__ __forceinline__ void sort_output_row(int32_t* oi, float* os, int n, uint64_t* ent, Fetch fetch) {
  if (n <= 1) return;
  const int P = next_pow2(n);
  for (int i = threadIdx.x; i < P; i += NTH) ent[i] = i < n ? comp_key(os[i], (uint32_t)oi[i]) : 0ull;
  __syncthreads();
  bitonic_sort_desc<NTH>(ent, P);
  for (int i = threadIdx.x; i < n; i += NTH) {
    uint32_t idx = comp_pos(ent[i]);
    oi[i] = (int32_t)idx;
    os[i] = fetch(idx);
  }
  __syncthreads();
}

// Exact top-k of row[0, n) by (score desc, index asc), written to oi/os
// (k entries, padded with (-1, -inf)). Plain most-significant-digit radix
// selection over the order keys: four 8-bit passes find the k-th key K*, then
// one ordered pass keeps every key > K* and the lowest-index keys == K*.
// Output order: ascending key index, or the total order when `sorted`.
template <int NTH>
__device__ __forceinline__ void radix_select_row_at(const float* row, int n, int k, int32_t* oi, float* os, bool sorted,
                                    uint8_t* lds);

// radix_select_row over keys [base, base + n) of a row whose key `base` is at
// row[0]: the written indices are shifted by `base`.
template <int NTH>
__device__ __forceinline__ void radix_select_row(const float* row, int n, int k, int32_t* oi, float* os, bool sorted,
                                 uint8_t* lds, int base = 0) {
  radix_select_row_at<NTH>(row, n, k, oi, os, sorted, lds);
  if (base != 0) {
    __threadfence_block();
    __syncthreads();
    for (int i = threadIdx.x; i < k; i += NTH)
      if (oi[i] >= 0) oi[i] += base;
  }
}

template <int NTH>
__device__ __forceinline__ void radix_select_row_at(const float* row, int n, int k, int32_t* oi, float* os, bool sorted,
                                    uint8_t* lds) {
  uint32_t* hist = reinterpret_cast<uint32_t*>(lds);
  uint32_t* tmp = hist + 256;                // 16 words
  uint64_t* ent = reinterpret_cast<uint64_t*>(lds + 256 * 4 + 64);
  const int tid = threadIdx.x;
  auto fetch = [&](uint32_t idx) { return row[idx]; };

  if (n <= k) {
    for (int i = tid; i < k; i += NTH) {
      if (i < n) {
        oi[i] = i;
        os[i] = row[i];
      } else {
        oi[i] = -1;
        os[i] = -__builtin_inff();
      }
    }
    if (sorted) {
      __threadfence_block();
      __syncthreads();
      sort_output_row<NTH>(oi, os, n, ent, fetch);
    }
    return;
  }

  uint32_t prefix = 0, pmask = 0, remaining = (uint32_t)k;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    for (int b = tid; b < 256; b += NTH) hist[b] = 0;
    __syncthreads();
    for (int i = tid; i < n; i += NTH) {
      uint32_t key = ord_key(row[i]);
      if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid < kWave) {
      uint32_t above = 0;
      int d = wave_threshold(hist, 256, remaining, &above);
      if (tid == 0) {
        tmp[8] = (uint32_t)d;
        tmp[9] = above;
      }
    }
    __syncthreads();
    const uint32_t d = tmp[8], above = tmp[9];
    __syncthreads();
    remaining -= above;
    prefix |= d << shift;
    pmask |= 0xFFu << shift;
  }
  const uint32_t kstar = prefix, need = remaining, ngt = (uint32_t)k - remaining;

  uint32_t run_gt = 0, run_eq = 0;
  for (int base = 0; base < n; base += NTH * 4) {
    const int i0 = base + tid * 4;
    float v[4];
    bool gt[4], eq[4];
    uint32_t cg = 0, ce = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = i0 + j;
      v[j] = i < n ? row[i] : 0.0f;
      uint32_t key = i < n ? ord_key(v[j]) : 0u;
      gt[j] = i < n && key > kstar;
      eq[j] = i < n && key == kstar;
      cg += gt[j];
      ce += eq[j];
    }
    uint32_t tot;
    uint32_t ex = block_scan_excl<NTH>((cg << 16) | ce, tmp, &tot);
    uint32_t g = run_gt + (ex >> 16), e = run_eq + (ex & 0xFFFFu);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (gt[j]) {
        uint32_t p = g + (e < need ? e : need);
        oi[p] = i0 + j;
        os[p] = v[j];
        ++g;
      } else if (eq[j]) {
        if (e < need) {
          uint32_t p = g + e;
          oi[p] = i0 + j;
          os[p] = v[j];
        }
        ++e;
      }
    }
    run_gt += tot >> 16;
    run_eq += tot & 0xFFFFu;
    if (run_gt >= ngt && run_eq >= need) break;  // block-uniform
  }
  if (sorted) {
    __threadfence_block();
    __syncthreads();
    sort_output_row<NTH>(oi, os, k, ent, fetch);
  }
}

}  // namespace lt
