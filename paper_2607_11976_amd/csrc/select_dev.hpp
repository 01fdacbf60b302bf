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

// The same network for P = NTH * E keys (E = 2..16): thread t holds keys
// [t * E, t * E + E) in registers for every stage whose stride is below E
// (the pairs of such a stage never leave a thread's block), and only the
// longer strides exchange through LDS: for 8192 keys on 1024 threads, 55
// LDS stages and 11 register passes instead of 91 LDS stages.
template <int NTH, int E, typename T>
__device__ __forceinline__ void bitonic_sort_desc_blk(T* a) {
  constexpr int P = NTH * E;
  constexpr int LOGE = E == 2 ? 1 : E == 4 ? 2 : E == 8 ? 3 : 4;
  static_assert((1 << LOGE) == E, "E must be 2, 4, 8 or 16");
  const int b0 = (int)threadIdx.x * E;
  T r[E];
  // strides E/2 .. 1 of the stage group of `size`, in registers
  auto reg_pass = [&](int size, int top) {
#pragma unroll
    for (int e = 0; e < E; ++e) r[e] = a[b0 + e];
#pragma unroll
    for (int sh = LOGE - 1; sh >= 0; --sh) {
      const int stride = 1 << sh;
      if (stride > top) continue;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        if ((e & stride) != 0) continue;
        const bool desc = ((b0 + e) & size) == 0;
        const T x = r[e], y = r[e + stride];
        if ((x < y) == desc) {
          r[e] = y;
          r[e + stride] = x;
        }
      }
    }
#pragma unroll
    for (int e = 0; e < E; ++e) a[b0 + e] = r[e];
    __syncthreads();
  };
  // sizes 2 .. E lie inside a thread's block
#pragma unroll
  for (int ls = 1; ls <= LOGE; ++ls) reg_pass(1 << ls, (1 << ls) >> 1);
  for (int size = 2 * E; size <= P; size <<= 1) {
    for (int stride = size >> 1; stride >= E; stride >>= 1) {
      for (int t = threadIdx.x; t < (P >> 1); t += NTH) {
        const int i = 2 * t - (t & (stride - 1));
        const int j = i + stride;
        const bool desc = (i & size) == 0;
        const T x = a[i], y = a[j];
        if ((x < y) == desc) {
          a[i] = y;
          a[j] = x;
        }
      }
      __syncthreads();
    }
    reg_pass(size, E >> 1);
  }
}

// bitonic_sort_desc with the register stages where P is 2 to 8 times NTH.
template <int NTH, typename T>
__device__ __forceinline__ void bitonic_sort_desc_fast(T* a, int P) {
  if (P == 8 * NTH) bitonic_sort_desc_blk<NTH, 8>(a);
  else if (P == 4 * NTH) bitonic_sort_desc_blk<NTH, 4>(a);
  else if (P == 2 * NTH) bitonic_sort_desc_blk<NTH, 2>(a);
  else bitonic_sort_desc<NTH>(a, P);
}

__host__ __device__ __forceinline__ int next_pow2(int n) {
  int p = 1;
  while (p < n) p <<= 1;
  return p;
}

// LDS layout of radix_select_row: a 256-bin histogram per wave (up to
// kRadixWaves waves), their sum, 32 words of exchange, then the sort entries.
constexpr int kRadixWaves = 8;
constexpr size_t kRadixTot = (size_t)kRadixWaves * 256 * 4;
constexpr size_t kRadixTmp = kRadixTot + 256 * 4;
constexpr size_t kRadixEnt = kRadixTmp + 32 * 4;

// Sort entries of radix_select_row: the output sort (k of them) and the keys
// of a digit prefix gathered in LDS once at most this many remain.
__host__ __device__ __forceinline__ int radix_collect_cap(int k) {
  const int p = next_pow2(k);
  return p < 4096 ? 4096 : p;
}
// LDS bytes radix_select_row needs for a given k.
__host__ __device__ __forceinline__ size_t radix_lds_bytes(int k) {
  return kRadixEnt + (size_t)radix_collect_cap(k) * 8;
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
// one pass writes every key > K* and the lowest-index keys == K*. Once at
// most radix_collect_cap(k) keys share the digits chosen so far (before any
// pass for rows that short), one last pass instead writes the keys above
// those digits and gathers the keys with them in LDS, which are sorted there
// by the total order; the best of them fill the remaining slots. Each wave
// streams a contiguous segment of the row (wave_stream) into its own
// histogram; the passes after the first test a key's prefix as a float range
// and the write pass compares floats with K*'s float (the order keys of the
// keys that pass are computed only for them); after each pass the wave also counts its keys
// above the pass's digit, so that after the last pass every wave knows how
// many keys > K* and == K* lie in the segments before its own, and the write
// pass places each hit without block barriers.
// Output order: ascending key index (after a gathering pass: the keys above
// the gathered digits in ascending key index, then the gathered ones in the
// total order), or the total order when `sorted`.
// pad = false: a row of n < k keys writes its n entries and nothing after.
template <int NTH>
__device__ __noinline__ void radix_select_row_at(const float* row, int n, int k, int32_t* oi, float* os, bool sorted,
                                                 uint8_t* lds, bool pad);

// radix_select_row over keys [base, base + n) of a row whose key `base` is at
// row[0]: the written indices are shifted by `base`.
template <int NTH>
__device__ __forceinline__ void radix_select_row(const float* row, int n, int k, int32_t* oi, float* os, bool sorted,
                                 uint8_t* lds, int base = 0, bool pad = true) {
  radix_select_row_at<NTH>(row, n, k, oi, os, sorted, lds, pad);
  if (base != 0) {
    __threadfence_block();
    __syncthreads();
    const int m = pad || n > k ? k : (n > 0 ? n : 0);
    for (int i = threadIdx.x; i < m; i += NTH)
      if (oi[i] >= 0) oi[i] += base;
  }
}

// Split fallback of one queued row whose visible keys [rs, rs + len) are cut
// into `chunks` chunks of `per` keys, chunk c = [kb, ke) scored into
// srow[kb, ke) by this block. The chunk's own exact top-k goes to the row's
// candidate region (cidx, cscore): chunk c's min(k, chunk length) entries
// after those of chunks 0..c-1, in ascending key order. The block that counts
// the row's last chunk (counter) selects the row from the candidates: the
// union of the chunks' top-k holds the row's top-k, in ascending key order,
// so positions order equal scores as key indices do. `flag`: one LDS word.
template <int NTH>
__device__ __forceinline__ void split_fallback_select(const float* srow, int rs, int len, int per, int chunks, int c,
                                                      int kb, int ke, int k, int32_t* cidx, float* cscore,
                                                      uint32_t* counter, int32_t* oi, float* os, bool sorted,
                                                      uint8_t* lds, int* flag) {
  auto clen = [&](int j) { return max(0, min(per, len - j * per)); };
  int off = 0;
  for (int j = 0; j < c; ++j) off += min(k, clen(j));
  radix_select_row<NTH>(srow + kb, ke - kb, k, cidx + off, cscore + off, false, lds, kb, false);
  // publish this chunk's candidates, then count it
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) *flag = atomicAdd(counter, 1u) == (uint32_t)(chunks - 1) ? 1 : 0;
  __syncthreads();
  if (!*flag) return;
  __threadfence();
  int u = 0;
  for (int j = 0; j < chunks; ++j) u += min(k, clen(j));
  radix_select_row_at<NTH>(cscore, u, k, oi, os, sorted, lds, true);
  __threadfence_block();
  __syncthreads();
  for (int i = threadIdx.x; i < k; i += NTH)
    if (oi[i] >= 0) oi[i] = cidx[oi[i]];
}

// Keys per lane of one streaming step, and the histogram passes (from the
// first) whose lanes of the most common bins add their counts with one
// atomic per bin. Measured on MI355X, one row of 262144 / 1M / 4M keys per
// 256-thread block: 0.41 / 1.5 / 5.7 ms with 16 keys and the next step in
// flight (0.72 / 2.6 / 10.1 ms before, with 32 plain loads per step and no
// look-ahead; 24 or 32 keys per step, no faster), 0.36 / 1.3 / 4.9 ms with
// the gathering pass in place of the last passes; without the grouped first
// pass the dense fallback of concentrated scores is 5% slower, four grouped
// bins in two passes slower too.
#ifndef LT_RADIX_UNROLL
#define LT_RADIX_UNROLL 16
#endif
#ifndef LT_RADIX_GROUP_PASSES
#define LT_RADIX_GROUP_PASSES 1
#endif
#ifndef LT_RADIX_GROUP_BINS
#define LT_RADIX_GROUP_BINS 1
#endif
constexpr int kRadixUnroll = LT_RADIX_UNROLL;

// One wave streams keys [s0, s1) of a row in steps of kWave * U keys (key
// s0 + j * kWave * U + u * kWave + lane in x[u] of step j). The loads of the
// next step are issued before the current step is processed, so that every
// step but the first finds its keys loaded while the previous one ran. The
// loads go through a buffer descriptor over the segment, whose range check
// turns the keys past s1 into zeros without a branch; body(c0, x) handles
// the step at key c0 (and tells the keys below s1 from those zeros itself,
// without branches: a step whose body branches on that makes the compiler
// wait for every load in flight). s0 and s1 are wave-uniform,
// s1 - s0 < 2^30.
template <int U, class Body>
__device__ __forceinline__ void wave_stream(const float* row, int s0, int s1, Body&& body) {
  constexpr int S = kWave * U;
  // the descriptor lives in scalar registers: the address and length are
  // made wave-uniform explicitly (a caller's arguments may sit in vector
  // registers, and a descriptor there would need a loop per load)
  const int len = __builtin_amdgcn_readfirstlane(s1 - s0);
  if (len <= 0) return;
  const uint64_t base = (uint64_t)(row + s0);
  const float* ubase = (const float*)((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)base) |
                                      (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(base >> 32)) << 32);
  // one descriptor per step (its base moves with the step, so every load
  // takes the lane's fixed offset plus an immediate)
  const int vo = lane_id() * 4;
  auto load = [&](int off, float (&x)[U]) {
    const int left = len - off;
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc((void*)(ubase + off), 0, left > 0 ? (int)((uint32_t)left * 4u) : 0, kBufferRaw);
#pragma unroll
    for (int u = 0; u < U; ++u)
      x[u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, vo + u * kWave * 4, 0, 0));
  };
  // two steps per trip and one exit, at the bottom (an exit between the
  // steps also makes the compiler wait for every load in flight): a step past
  // s1 loads only zeros and its body finds no key below s1
  float xa[U], xb[U];
  load(0, xa);
  for (int off = 0; off < len; off += 2 * S) {
    load(off + S, xb);
    body(s0 + off, xa);
    load(off + 2 * S, xa);
    body(s0 + off + S, xb);
  }
}

// radix_select_row_at of a row of n <= k keys: every key is taken (a
// function of its own: inside the selection its branch made the compiler
// wait for every load in flight in the streaming loops).
template <int NTH>
__device__ __noinline__ void radix_copy_short_row(const float* row, int n, int k, int32_t* oi, float* os, bool sorted,
                                                  uint8_t* lds, bool pad) {
  uint64_t* ent = reinterpret_cast<uint64_t*>(lds + kRadixEnt);
  const int tid = threadIdx.x;
  auto fetch = [&](uint32_t idx) { return row[idx]; };
  for (int i = tid; i < k; i += NTH) {
    if (i < n) {
      oi[i] = i;
      os[i] = row[i];
    } else if (pad) {
      oi[i] = -1;
      os[i] = -__builtin_inff();
    }
  }
  if (sorted) {
    __threadfence_block();
    __syncthreads();
    sort_output_row<NTH>(oi, os, n, ent, fetch);
  }
}

// Not inlined: the callers inline it after a register-heavy scan, and a
// separate allocation keeps its unrolled loads from spilling the scan.
template <int NTH>
__device__ __noinline__ void radix_select_row_at(const float* row, int n, int k, int32_t* oi, float* os, bool sorted,
                                                 uint8_t* lds, bool pad) {
  constexpr int NW = NTH / kWave, U = kRadixUnroll;
  static_assert(NW <= kRadixWaves, "one histogram per wave");
  static_assert(NW >= 4, "segments of fewer than 2^30 keys");
  // the sizes and flags are the same in every lane (arguments arrive in
  // vector registers): branches on them stay scalar, which keeps the loads
  // of the streaming loops in flight across their steps
  n = __builtin_amdgcn_readfirstlane(n);
  k = __builtin_amdgcn_readfirstlane(k);
  sorted = __builtin_amdgcn_readfirstlane((int)sorted) != 0;
  pad = __builtin_amdgcn_readfirstlane((int)pad) != 0;
  uint32_t* hist = reinterpret_cast<uint32_t*>(lds);              // [NW][256]
  uint32_t* tot = reinterpret_cast<uint32_t*>(lds + kRadixTot);   // [256]
  uint32_t* tmp = reinterpret_cast<uint32_t*>(lds + kRadixTmp);   // [32]
  uint64_t* ent = reinterpret_cast<uint64_t*>(lds + kRadixEnt);
  const int tid = threadIdx.x, l = lane_id(), wave = tid / kWave;
  uint32_t* hw = hist + wave * 256;
  auto fetch = [&](uint32_t idx) { return row[idx]; };

  if (n <= k) {
    radix_copy_short_row<NTH>(row, n, k, oi, os, sorted, lds, pad);
    return;
  }
  // this wave's segment [s0, s1) of the row
  const int seg = ((n + NW - 1) / NW + kWave - 1) / kWave * kWave;
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  const int s0 = min(wv * seg, n), s1 = min(s0 + seg, n);

  uint32_t prefix = 0, pmask = 0, remaining = (uint32_t)k;
  uint32_t gbefore = 0;  // this wave's keys above the digits chosen so far (wave-uniform)
  uint32_t eqw = 0;      // this wave's keys == K* (after the last pass)
  uint32_t inbin = (uint32_t)n;  // keys with the digits chosen so far
  const uint32_t cap = (uint32_t)radix_collect_cap(k);
  bool collected = false;
  for (int pass = 0; pass < 4; ++pass) {
    if (inbin <= cap) {  // wave-uniform
      // Few keys left with the chosen digits: one last pass writes the keys
      // above them to the output (after those of lower waves, counted by
      // gbefore) and gathers them in LDS as (key, index) sort entries; the
      // best `remaining` of those, by the total order, fill the last slots.
      if (l == 0) tmp[wave] = gbefore;
      if (tid == 0) tmp[18] = 0u;
      __syncthreads();
      uint32_t g = 0;
      for (int w = 0; w < wv; ++w) g += tmp[w];
      wave_stream<U>(row, s0, s1, [&](int c0, const float (&x)[U]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int i = c0 + u * kWave + l;
          const bool v = i < s1;
          const uint32_t kp = ord_key(x[u]) & pmask;
          const bool ab = v & (kp > prefix), in = v & (kp == prefix);
          const uint64_t ma = __ballot(ab), mi = __ballot(in);
          if (ab) {
            const uint32_t p = g + mbcnt64(ma);
            oi[p] = i;
            os[p] = x[u];
          }
          g += (uint32_t)__popcll(ma);
          if (mi != 0) {  // wave-uniform: one slot reservation for the wave's keys
            const int lead = (int)__builtin_ctzll(mi);
            uint32_t base = 0u;
            if (l == lead) base = atomicAdd(&tmp[18], (uint32_t)__popcll(mi));
            base = (uint32_t)__builtin_amdgcn_readlane((int)base, lead);
            const uint32_t sl = base + mbcnt64(mi);
            if (in && sl < cap) ent[sl] = comp_key(x[u], (uint32_t)i);
          }
        }
      });
      __syncthreads();
      const uint32_t cnt = min(tmp[18], cap);
      const int P = next_pow2(cnt < 1u ? 1 : (int)cnt);
      for (int j = (int)cnt + tid; j < P; j += NTH) ent[j] = 0ull;
      __syncthreads();
      bitonic_sort_desc<NTH>(ent, P);
      const uint32_t first = (uint32_t)k - remaining;
      for (uint32_t j = tid; j < remaining; j += NTH) {
        const uint32_t idx = comp_pos(ent[j]);
        oi[first + j] = (int32_t)idx;
        os[first + j] = row[idx];
      }
      collected = true;
      break;
    }
    const int shift = 24 - 8 * pass;
    for (int b = tid; b < NW * 256; b += NTH) hist[b] = 0;
    __syncthreads();
    // GROUP (the first passes): concentrated scores share their leading
    // bytes, so the lanes of the few most common bins add their counts with
    // one atomic per bin
    auto hist_pass = [&]<bool GROUP>() {
      wave_stream<U>(row, s0, s1, [&](int c0, const float (&x)[U]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
          // (bool & bool: a short-circuit && would branch)
          const bool v = c0 + u * kWave + l < s1;
          const uint32_t key = ord_key(x[u]);
          const uint32_t b = (key >> shift) & 255u;
          bool in = v & ((key & pmask) == prefix);
          if constexpr (GROUP) {
            uint64_t left = __ballot(in);
#pragma unroll
            for (int g = 0; g < LT_RADIX_GROUP_BINS; ++g) {
              if (left == 0) break;
              const uint32_t bg = __builtin_amdgcn_readlane(b, __builtin_ctzll(left));
              const uint64_t mg = __ballot(in && b == bg);
              if (l == (int)__builtin_ctzll(mg)) atomicAdd(&hw[bg], (uint32_t)__popcll(mg));
              in = in && b != bg;
              left &= ~mg;
            }
          }
          if (in) atomicAdd(&hw[b], 1u);
        }
      });
    };
    if (pass < LT_RADIX_GROUP_PASSES) {
      hist_pass.template operator()<true>();
    } else if (prefix == 0u) {
      hist_pass.template operator()<false>();
    } else {
      // a prefix other than 0 (the NaN key) spans the order keys of the
      // floats in [lo, hi]: two compares find the keys of the prefix, and
      // only their digits are computed (keys past +inf are NaN codes no
      // score maps to; below +0 lies -0's unused key, so the top of a range
      // that ends there is the largest negative float)
      const uint32_t lk = prefix < 0x007FFFFFu ? 0x007FFFFFu : prefix;
      uint32_t hk = prefix | ~pmask;
      hk = hk > 0xFF800000u ? 0xFF800000u : hk == 0x7FFFFFFFu ? 0x7FFFFFFEu : hk;
      const float lo = ord_inv(lk), hi = ord_inv(hk);
      wave_stream<U>(row, s0, s1, [&](int c0, const float (&x)[U]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const bool in = (c0 + u * kWave + l < s1) & (x[u] >= lo) & (x[u] <= hi);
          if (in) atomicAdd(&hw[(ord_key(x[u]) >> shift) & 255u], 1u);
        }
      });
    }
    __syncthreads();
    for (int b = tid; b < 256; b += NTH) {
      uint32_t t = 0;
      for (int w = 0; w < NW; ++w) t += hist[w * 256 + b];
      tot[b] = t;
    }
    __syncthreads();
    if (tid < kWave) {
      uint32_t above = 0;
      int d = wave_threshold(tot, 256, remaining, &above);
      if (tid == 0) {
        tmp[16] = (uint32_t)d;
        tmp[17] = above;
      }
    }
    __syncthreads();
    // (read into scalar registers: the digit chooses the next pass's loop,
    // and a choice the compiler cannot see as wave-uniform becomes a masked
    // branch around loops whose loads then all wait for each other)
    const uint32_t d = __builtin_amdgcn_readfirstlane(tmp[16]), above = __builtin_amdgcn_readfirstlane(tmp[17]);
    const uint32_t nbin = __builtin_amdgcn_readfirstlane(tot[d]);
    // this wave's keys of the current prefix in bins above d (and == d)
    uint32_t mine = 0;
    for (int b = l; b < 256; b += kWave) mine += (uint32_t)b > d ? hw[b] : 0u;
    gbefore += wave_sum(mine);
    if (pass == 3) eqw = hw[d];
    __syncthreads();
    remaining -= above;
    prefix |= d << shift;
    pmask |= 0xFFu << shift;
    inbin = nbin;
  }
  if (collected) {  // block-uniform
    if (sorted) {
      __threadfence_block();
      __syncthreads();
      sort_output_row<NTH>(oi, os, k, ent, fetch);
    }
    return;
  }
  const uint32_t kstar = prefix, need = remaining;
  if (l == 0) {
    tmp[wave] = gbefore;
    tmp[8 + wave] = eqw;
  }
  __syncthreads();
  uint32_t g = 0, e = 0, cg = 0, ce = 0;
  for (int w = 0; w < NW; ++w) {
    if (w < wave) {
      g += tmp[w];
      e += tmp[8 + w];
    }
  }
  cg = tmp[wave];
  ce = tmp[8 + wave];
  __syncthreads();
  // a key > K* goes after the keys > K* and the taken keys == K* of lower
  // index; a key == K* is taken while fewer than `need` of lower index were
  // for K* other than the NaN key, the float K with that key: key > K* and
  // key == K* are the float compares x > K and x == K (NaN fails both; -0
  // and +0 share a key and compare equal); for the NaN key, key > K* is
  // "not NaN" and key == K* is "NaN"
  const float kf = ord_inv(kstar);
  auto write_pass = [&]<bool KNAN>() {
    wave_stream<U>(row, s0, s1, [&](int c0, const float (&x)[U]) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = c0 + u * kWave + l;
        const bool v = i < s1;
        const bool gt = v & (KNAN ? x[u] == x[u] : x[u] > kf), eq = v & (KNAN ? x[u] != x[u] : x[u] == kf);
        const uint64_t mg = __ballot(gt), me = __ballot(eq);
        if ((mg | me) == 0) continue;
        const uint32_t rg = g + mbcnt64(mg), re = e + mbcnt64(me);
        if (gt) {
          const uint32_t p = rg + (re < need ? re : need);
          oi[p] = i;
          os[p] = x[u];
        } else if (eq && re < need) {
          const uint32_t p = rg + re;
          oi[p] = i;
          os[p] = x[u];
        }
        g += (uint32_t)__popcll(mg);
        e += (uint32_t)__popcll(me);
      }
    });
  };
  if (cg != 0 || (ce != 0 && e < need)) {  // wave-uniform
    if (kstar == 0u) write_pass.template operator()<true>();
    else write_pass.template operator()<false>();
  }
  if (sorted) {
    __threadfence_block();
    __syncthreads();
    sort_output_row<NTH>(oi, os, k, ent, fetch);
  }
}

}  // namespace lt
