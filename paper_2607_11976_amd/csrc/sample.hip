// Sample key lists (sec. 3.2 "Sampling"). Every launch scores its sample
// from a list of key indices in the workspace; entries < 0 are holes that
// every consumer skips. The list comes from one of:
//  * the random stratified sample (k_sample_list);
//  * a caller's list, cleaned so that it holds distinct in-range keys
//    (k_list_clean) -- the initial threshold is only a lower bound of the
//    row's k-th score if every sampled score is one of the row's scores,
//    counted once;
//  * the previous chunk's top-k (lt_sample_from_topk): the keys that occur
//    most often there, found by a most-significant-digit radix selection over
//    the per-key occurrence counts.
#include <algorithm>

#include "internal.hpp"
#include "select_dev.hpp"

namespace lt {

__global__ __launch_bounds__(256) void k_sample_list(int32_t* list, int ns, int nk, int blk, uint64_t seed) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < ns) list[i] = sample_key(i, ns, nk, blk, seed);
}

hipError_t launch_sample_list(int32_t* list, int ns, int nk, int blk, uint64_t seed, hipStream_t st) {
  if (ns <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_sample_list, dim3((ns + 255) / 256), dim3(256), 0, st, list, ns, nk, blk, seed);
  return hipGetLastError();
}

// One block. Fast path: when the in-range entries already come in strictly
// ascending order (the previous-chunk sampler writes such lists), the list
// only needs its out-of-range entries turned into holes. Otherwise sort it
// ascending (as the descending order of ~key, which puts the out-of-range
// entries, mapped to 0, last), keep the first of each run of equal keys, and
// write holes (-1) for everything else.
constexpr int kCleanThreads = 1024;

__global__ __launch_bounds__(kCleanThreads) void k_list_clean(const int32_t* in, int ns, int nk, int32_t* out) {
  extern __shared__ __align__(16) uint32_t a[];
  __shared__ int wave_last[kCleanThreads / kWave];
  const int tid = threadIdx.x, l = lane_id(), w = tid / kWave;
  // thread t checks its own segment; segments are ordered by t
  const int seg = (ns + kCleanThreads - 1) / kCleanThreads;
  const int lo = tid * seg, hi = min(lo + seg, ns);
  int first = -1, last = -1;
  bool ok = true;
  for (int i = lo; i < hi; ++i) {
    const int v = in[i];
    if (v < 0 || v >= nk) continue;
    if (first < 0) first = v;
    ok = ok && v > last;
    last = v;
  }
  // largest in-range entry of all earlier segments: exclusive max-scan of `last`
  int run = last;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int t = __shfl_up(run, off, kWave);
    if (l >= off) run = max(run, t);
  }
  if (l == kWave - 1) wave_last[w] = run;
  int before = __shfl_up(run, 1, kWave);
  if (l == 0) before = -1;
  __syncthreads();
  for (int i = 0; i < w; ++i) before = max(before, wave_last[i]);
  ok = ok && (first < 0 || first > before);
  if (__syncthreads_and(ok)) {
    for (int i = tid; i < ns; i += kCleanThreads) {
      const int v = in[i];
      out[i] = (v >= 0 && v < nk) ? v : -1;
    }
    return;
  }
  const int P = next_pow2(ns);
  for (int i = tid; i < P; i += kCleanThreads) {
    const int v = i < ns ? in[i] : -1;
    a[i] = (v >= 0 && v < nk) ? ~(uint32_t)v : 0u;
  }
  __syncthreads();
  bitonic_sort_desc<kCleanThreads>(a, P);
  for (int i = tid; i < ns; i += kCleanThreads) {
    const uint32_t x = a[i];
    const bool keep = x != 0u && (i == 0 || a[i - 1] != x);
    out[i] = keep ? (int32_t)~x : -1;
  }
}

hipError_t launch_list_clean(const int32_t* in, int ns, int nk, int32_t* out, hipStream_t st) {
  if (ns <= 0) return hipSuccess;
  const size_t lds = (size_t)next_pow2(ns) * 4;
  if (lds > 65536)
    (void)hipFuncSetAttribute((const void*)k_list_clean, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  hipLaunchKernelGGL(k_list_clean, dim3(1), dim3(kCleanThreads), lds, st, in, ns, nk, out);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Previous-chunk sample. The order is (count desc, key asc); the selected set
// is the first sample_size keys of it that have count >= 1. The count c* of
// the last selected key is found from histograms of the counts: when fewer
// than sample_size keys can reach a count of 2047 (entries / 2047 <
// sample_size, known on the host), one histogram of the counts clamped at
// 2047 gives c* directly; otherwise c* is found digit by digit (11 + 11 + 10
// bits, most significant first), each pass histogramming the digit of every
// count that matches the digits fixed so far. The last block of each
// histogram launch is followed by a one-wave pick of the digit (where the
// running total from the top reaches the number still wanted). Then the keys with count > c*
// and the first `need` keys with count == c* (ascending key order, count >=
// 1) are compacted in key order.
// ---------------------------------------------------------------------------
constexpr int kFreqThreads = 1024;
constexpr int kFreqBins = 2048;
constexpr int kFreqMaxBlocks = 1024;
constexpr int kFreqClampPass = 3;  // the single pass over counts clamped at kFreqBins - 1

struct FreqState {
  uint32_t prefix;  // digits fixed so far (the clamped pass: c* itself)
  uint32_t mask;    // their bit mask
  uint32_t want;    // keys still to take at or below the fixed prefix
  uint32_t above;   // keys whose count exceeds every candidate of the prefix
};

__host__ __device__ constexpr int freq_shift(int pass) { return pass == 0 ? 21 : (pass == 1 ? 10 : 0); }
__host__ __device__ constexpr int freq_bits(int pass) { return pass == 2 ? 10 : 11; }

__global__ __launch_bounds__(kFreqThreads) void k_freq_zero(uint32_t* counts, int nk, uint32_t* hist,
                                                             FreqState* fs, int ns) {
  const int64_t stride = (int64_t)gridDim.x * kFreqThreads;
  for (int64_t i = (int64_t)blockIdx.x * kFreqThreads + threadIdx.x; i < nk; i += stride) counts[i] = 0u;
  if (blockIdx.x == 0) {
    for (int i = threadIdx.x; i < 4 * kFreqBins; i += kFreqThreads) hist[i] = 0u;
    if (threadIdx.x == 0) *fs = FreqState{0u, 0u, (uint32_t)ns, 0u};
  }
}

__global__ __launch_bounds__(kFreqThreads) void k_freq_count(const int32_t* prev, int64_t ld, int rows, int pk,
                                                              int nk, uint32_t* counts) {
  const int64_t total = (int64_t)rows * pk;
  const int64_t stride = (int64_t)gridDim.x * kFreqThreads;
  for (int64_t e = (int64_t)blockIdx.x * kFreqThreads + threadIdx.x; e < total; e += stride) {
    const int64_t t = e / pk;
    const int v = prev[t * ld + (e - t * pk)];
    if (v >= 0 && v < nk) atomicAdd(&counts[v], 1u);
  }
}

// One wave picks the digit of `pass` from its histogram h: lane l owns digits
// [l * per, (l + 1) * per), read once into registers.
__device__ void freq_pick(int pass, const uint32_t* h, FreqState* fs) {
  constexpr int kPer = kFreqBins / kWave;
  const int l = lane_id();
  const int nb = pass == kFreqClampPass ? kFreqBins : 1 << freq_bits(pass), per = nb / kWave;
  uint32_t hr[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) hr[j] = j < per ? h[l * per + j] : 0u;
  uint32_t loc = 0;
#pragma unroll
  for (int j = 0; j < kPer; ++j) loc += hr[j];
  const uint32_t want = fs->want;
  uint32_t run = wave_suffix_sum_excl(loc);  // matching keys with a digit above this lane's range
  int dig = -1;
  uint32_t gt = 0;
#pragma unroll
  for (int j = kPer - 1; j >= 0; --j) {
    if (j >= per) continue;
    const uint32_t nxt = run + hr[j];
    if (run < want && nxt >= want) {
      dig = l * per + j;
      gt = run;
    }
    run = nxt;
  }
  // no crossing: fewer matching keys than wanted (only when num_keys is below
  // the sample size): take all of them, i.e. go on with digit 0
  const uint64_t found = __ballot(dig >= 0);
  if (!found) {
    const uint32_t total = wave_sum(loc);
    const uint32_t h0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)hr[0]);  // lane 0 holds digit 0
    if (l == 0) {
      dig = 0;
      gt = total - h0;
    }
  }
  const bool writer = found ? dig >= 0 : l == 0;
  if (writer) {
    FreqState s = *fs;
    if (pass == kFreqClampPass) {
      s.prefix = (uint32_t)dig;
      s.mask = ~0u;
    } else {
      const int shift = freq_shift(pass);
      const uint32_t dmask = (1u << freq_bits(pass)) - 1u;
      s.prefix |= (uint32_t)dig << shift;
      s.mask |= dmask << shift;
    }
    s.above += gt;
    s.want = want - gt;
    *fs = s;
  }
}

// Histogram add of digit dg (when match) to the LDS histogram h. Most counts
// are small: one LDS add per wave for each of the digits 0..15, a lane's own
// add for the others.
__device__ __forceinline__ void freq_hist_add(uint32_t* h, bool match, uint32_t dg, int l) {
#pragma unroll
  for (uint32_t b = 0; b < 16u; ++b) {
    const uint64_t mk = __ballot(match && dg == b);
    if (l == 0 && mk) atomicAdd(&h[b], (uint32_t)__popcll(mk));
  }
  if (match && dg >= 16u) atomicAdd(&h[dg], 1u);
}

// One wave picks the digit of a pass, in a launch of its own: a release fence
// in every histogram block (so that the last one could pick) writes back the
// L2s and cost more than the launch.
__global__ __launch_bounds__(kWave) void k_freq_pick(int pass, const uint32_t* hist, FreqState* fs) {
  freq_pick(pass, hist + pass * kFreqBins, fs);
}

__global__ __launch_bounds__(kFreqThreads) void k_freq_hist(const uint32_t* counts, int nk, int pass,
                                                             FreqState* fs, uint32_t* hist) {
  __shared__ uint32_t h[kFreqBins];
  for (int i = threadIdx.x; i < kFreqBins; i += kFreqThreads) h[i] = 0u;
  __syncthreads();
  const bool clamp = pass == kFreqClampPass;
  const uint32_t prefix = clamp ? 0u : fs->prefix, mask = clamp ? 0u : fs->mask;
  const int shift = clamp ? 0 : freq_shift(pass);
  const uint32_t dmask = clamp ? ~0u : (1u << freq_bits(pass)) - 1u;
  const int l = lane_id();
  const int64_t stride = (int64_t)gridDim.x * kFreqThreads;
  const int64_t span = ((int64_t)nk + kFreqThreads - 1) / kFreqThreads * kFreqThreads;
  for (int64_t s = (int64_t)blockIdx.x * kFreqThreads + threadIdx.x; s < span; s += stride) {
    const uint32_t c = s < nk ? counts[s] : 0u;
    const bool match = s < nk && (c & mask) == prefix;
    const uint32_t dg = min((c >> shift) & dmask, (uint32_t)(kFreqBins - 1));
    freq_hist_add(h, match, dg, l);
  }
  __syncthreads();
  uint32_t* hp = hist + pass * kFreqBins;
  for (int i = threadIdx.x; i < kFreqBins; i += kFreqThreads)
    if (h[i]) atomicAdd(hp + i, h[i]);
}

// Counting in LDS for key arrays up to kFreqLdsMaxKeys: block (r, ch) counts
// the keys of range r (kFreqRange keys) among entry chunk ch and stores the
// counts to part[ch][key]; no global atomics (random global atomic adds from
// the whole GPU ran at about 10 per ns). Block (0, 0) also clears the
// histograms and the selection state.
constexpr int kFreqRange = 16384;
constexpr int kFreqParts = 32;
constexpr int kFreqLdsMaxKeys = 262144;

__global__ __launch_bounds__(kFreqThreads) void k_freq_count_lds(const int32_t* prev, int64_t ld, int rows, int pk,
                                                                  int nk, uint32_t* part, uint32_t* hist,
                                                                  FreqState* fs, int ns) {
  __shared__ uint32_t c[kFreqRange];
  const int lo = blockIdx.x * kFreqRange, n = min(kFreqRange, nk - lo), ch = blockIdx.y, nch = gridDim.y;
  if (blockIdx.x == 0 && ch == 0) {
    for (int i = threadIdx.x; i < 4 * kFreqBins; i += kFreqThreads) hist[i] = 0u;
    if (threadIdx.x == 0) *fs = FreqState{0u, 0u, (uint32_t)ns, 0u};
  }
  for (int i = threadIdx.x; i < kFreqRange; i += kFreqThreads) c[i] = 0u;
  __syncthreads();
  // rows * pk < 2^31 (checked on the host); entry e = row t, column j, the
  // thread's (t, j) advanced by the stride without a division per entry
  const uint32_t upk = (uint32_t)pk, total = (uint32_t)rows * upk, per = (total + nch - 1) / nch;
  const uint32_t e0 = (uint32_t)ch * per, e1 = min(e0 + per, total);
  const uint32_t dt = kFreqThreads / upk, dj = kFreqThreads % upk;
  uint32_t t = (e0 + threadIdx.x) / upk, j = (e0 + threadIdx.x) - t * upk;
  auto step = [&]() {
    t += dt;
    j += dj;
    if (j >= upk) {
      j -= upk;
      ++t;
    }
  };
  // eight loads in flight per thread, then their counts
  constexpr int kU = 8;
  uint32_t e = e0 + threadIdx.x;
  for (; e + (kU - 1) * kFreqThreads < e1; e += kU * kFreqThreads) {
    int v[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      v[u] = prev[(int64_t)t * ld + j];
      step();
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int x = v[u] - lo;
      if (x >= 0 && x < n) atomicAdd(&c[x], 1u);
    }
  }
  for (; e < e1; e += kFreqThreads) {
    const int x = prev[(int64_t)t * ld + j] - lo;
    if (x >= 0 && x < n) atomicAdd(&c[x], 1u);
    step();
  }
  __syncthreads();
  for (int i = threadIdx.x; i < n; i += kFreqThreads) part[(int64_t)ch * nk + lo + i] = c[i];
}

// counts[key] = sum of the chunks' counts; with `clamp`, also the histogram
// of the counts clamped at kFreqBins - 1.
__global__ __launch_bounds__(kFreqThreads) void k_freq_merge(const uint32_t* part, int nparts, int nk, bool clamp,
                                                              uint32_t* counts, uint32_t* hist) {
  __shared__ uint32_t h[kFreqBins];
  for (int i = threadIdx.x; i < kFreqBins; i += kFreqThreads) h[i] = 0u;
  __syncthreads();
  const int l = lane_id();
  const int64_t stride = (int64_t)gridDim.x * kFreqThreads;
  const int64_t span = ((int64_t)nk + kFreqThreads - 1) / kFreqThreads * kFreqThreads;
  for (int64_t s = (int64_t)blockIdx.x * kFreqThreads + threadIdx.x; s < span; s += stride) {
    uint32_t c = 0;
    if (s < nk) {
      uint32_t c4[4] = {0u, 0u, 0u, 0u};
      int ch = 0;
      for (; ch + 4 <= nparts; ch += 4)
#pragma unroll
        for (int u = 0; u < 4; ++u) c4[u] += part[(int64_t)(ch + u) * nk + s];
      for (; ch < nparts; ++ch) c4[0] += part[(int64_t)ch * nk + s];
      c = c4[0] + c4[1] + c4[2] + c4[3];
      counts[s] = c;
    }
    if (clamp) freq_hist_add(h, s < nk, min(c, (uint32_t)(kFreqBins - 1)), l);
  }
  if (!clamp) return;
  __syncthreads();
  uint32_t* hp = hist + kFreqClampPass * kFreqBins;
  for (int i = threadIdx.x; i < kFreqBins; i += kFreqThreads)
    if (h[i]) atomicAdd(hp + i, h[i]);
}

// Selected-key flags of one key: count > c*, or the tie rank decides.
struct FreqSel {
  uint32_t cstar, need;
  __device__ bool gt(uint32_t c) const { return c > cstar && c > 0u; }
  __device__ bool eq(uint32_t c) const { return c == cstar && cstar > 0u; }
};

__device__ __forceinline__ FreqSel freq_sel(const FreqState* fs) {
  const FreqState s = *fs;
  return FreqSel{s.prefix, s.prefix > 0u ? s.want : 0u};
}

__global__ __launch_bounds__(kFreqThreads) void k_freq_blocks(const uint32_t* counts, int nk, int chunk,
                                                               const FreqState* fs, uint32_t* bc) {
  __shared__ uint32_t tmp[kFreqThreads / kWave];
  const FreqSel f = freq_sel(fs);
  const int64_t lo = (int64_t)blockIdx.x * chunk, hi = std::min<int64_t>(lo + chunk, nk);
  uint32_t g = 0, e = 0;
  for (int64_t s = lo + threadIdx.x; s < hi; s += kFreqThreads) {
    const uint32_t c = counts[s];
    g += f.gt(c);
    e += f.eq(c);
  }
  uint32_t tg, te;
  (void)block_scan_excl<kFreqThreads>(g, tmp, &tg);
  (void)block_scan_excl<kFreqThreads>(e, tmp, &te);
  if (threadIdx.x == 0) {
    bc[2 * blockIdx.x] = tg;
    bc[2 * blockIdx.x + 1] = te;
  }
}

__global__ __launch_bounds__(kFreqThreads) void k_freq_emit(const uint32_t* counts, int nk, int chunk,
                                                             const FreqState* fs, const uint32_t* bc, int ns,
                                                             int32_t* out) {
  __shared__ uint32_t tmp[kFreqThreads / kWave];
  const FreqSel f = freq_sel(fs);
  // selected keys and ties before this block
  uint32_t g0 = 0, e0 = 0;
  for (int b = threadIdx.x; b < (int)blockIdx.x; b += kFreqThreads) {
    g0 += bc[2 * b];
    e0 += bc[2 * b + 1];
  }
  uint32_t run_g, run_e;
  (void)block_scan_excl<kFreqThreads>(g0, tmp, &run_g);
  (void)block_scan_excl<kFreqThreads>(e0, tmp, &run_e);
  const int64_t lo = (int64_t)blockIdx.x * chunk, hi = std::min<int64_t>(lo + chunk, nk);
  for (int64_t base = lo; base < hi; base += kFreqThreads) {
    const int64_t s = base + threadIdx.x;
    const uint32_t c = s < hi ? counts[s] : 0u;
    const bool g = s < hi && f.gt(c), e = s < hi && f.eq(c);
    uint32_t tot;
    const uint32_t ex = block_scan_excl<kFreqThreads>(((uint32_t)g << 16) | (uint32_t)e, tmp, &tot);
    const uint32_t gi = run_g + (ex >> 16), ei = run_e + (ex & 0xFFFFu);
    // position = selected keys before s: every earlier count > c*, and the
    // earlier ties up to `need`
    if (g) out[gi + std::min(ei, f.need)] = (int32_t)s;
    if (e && ei < f.need) out[gi + ei] = (int32_t)s;
    run_g += tot >> 16;
    run_e += tot & 0xFFFFu;
  }
  // padding after the last selected key
  const FreqState st = *fs;
  const uint32_t nsel = st.above + (st.prefix > 0u ? st.want : 0u);
  const int64_t stride = (int64_t)gridDim.x * kFreqThreads;
  for (int64_t p = nsel + (int64_t)blockIdx.x * kFreqThreads + threadIdx.x; p < ns; p += stride) out[p] = -1;
}

size_t freq_workspace_bytes(int nk) {
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t parts = nk <= kFreqLdsMaxKeys ? up((size_t)kFreqParts * nk * 4) : 0;
  return up((size_t)nk * 4) + up(4 * kFreqBins * 4) + up(sizeof(FreqState)) + up(2 * kFreqMaxBlocks * 4) + parts;
}

hipError_t launch_sample_from_topk(const int32_t* prev, int64_t ld, int rows, int pk, int nk, int ns,
                                   int32_t* out, void* ws, hipStream_t st) {
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  uint8_t* p = static_cast<uint8_t*>(ws);
  uint32_t* counts = reinterpret_cast<uint32_t*>(p);
  p += up((size_t)nk * 4);
  uint32_t* hist = reinterpret_cast<uint32_t*>(p);
  p += up(4 * kFreqBins * 4);
  FreqState* fs = reinterpret_cast<FreqState*>(p);
  p += up(sizeof(FreqState));
  uint32_t* bc = reinterpret_cast<uint32_t*>(p);
  p += up(2 * kFreqMaxBlocks * 4);
  uint32_t* part = reinterpret_cast<uint32_t*>(p);

  const int sweep = (int)std::min<int64_t>(256, std::max<int64_t>(1, ((int64_t)nk + 4095) / 4096));
  int nb = (int)std::min<int64_t>(kFreqMaxBlocks, std::max<int64_t>(1, ((int64_t)nk + 4095) / 4096));
  const int chunk = (int)((((int64_t)nk + nb - 1) / nb + kFreqThreads - 1) / kFreqThreads * kFreqThreads);
  const int64_t entries = (int64_t)rows * pk;
  const int cgrid = (int)std::min<int64_t>(1024, std::max<int64_t>(1, (entries + kFreqThreads - 1) / kFreqThreads));

  // fewer than ns keys can reach a count of kFreqBins - 1: one clamped pass
  const bool clamp = entries / (kFreqBins - 1) < ns;
  if (nk > 0 && nk <= kFreqLdsMaxKeys) {
    // about 128 counting blocks; the merge reads each key's chunk counts
    // with one thread per key
    const int ranges = (nk + kFreqRange - 1) / kFreqRange;
    const int nparts = std::max(1, std::min(kFreqParts, 128 / ranges));
    const int mgrid = (nk + kFreqThreads - 1) / kFreqThreads;
    hipLaunchKernelGGL(k_freq_count_lds, dim3(ranges, nparts), dim3(kFreqThreads), 0, st, prev, ld, rows, pk, nk,
                       part, hist, fs, ns);
    hipLaunchKernelGGL(k_freq_merge, dim3(mgrid), dim3(kFreqThreads), 0, st, part, nparts, nk, clamp, counts, hist);
    if (clamp) hipLaunchKernelGGL(k_freq_pick, dim3(1), dim3(kWave), 0, st, kFreqClampPass, hist, fs);
  } else {
    hipLaunchKernelGGL(k_freq_zero, dim3(sweep), dim3(kFreqThreads), 0, st, counts, nk, hist, fs, ns);
    if (entries > 0)
      hipLaunchKernelGGL(k_freq_count, dim3(cgrid), dim3(kFreqThreads), 0, st, prev, ld, rows, pk, nk, counts);
    if (clamp) {
      hipLaunchKernelGGL(k_freq_hist, dim3(sweep), dim3(kFreqThreads), 0, st, counts, nk, kFreqClampPass, fs, hist);
      hipLaunchKernelGGL(k_freq_pick, dim3(1), dim3(kWave), 0, st, kFreqClampPass, hist, fs);
    }
  }
  if (!clamp)
    for (int pass = 0; pass < 3; ++pass) {
      hipLaunchKernelGGL(k_freq_hist, dim3(sweep), dim3(kFreqThreads), 0, st, counts, nk, pass, fs, hist);
      hipLaunchKernelGGL(k_freq_pick, dim3(1), dim3(kWave), 0, st, pass, hist, fs);
    }
  hipLaunchKernelGGL(k_freq_blocks, dim3(nb), dim3(kFreqThreads), 0, st, counts, nk, chunk, fs, bc);
  hipLaunchKernelGGL(k_freq_emit, dim3(nb), dim3(kFreqThreads), 0, st, counts, nk, chunk, fs, bc, ns, out);
  return hipGetLastError();
}

}  // namespace lt
