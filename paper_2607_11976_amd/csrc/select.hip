// Selection-side kernels: per-row range from the sample, the scores-in
// filter scan, the final select, the exact fallback and plain radix select.
#include "internal.hpp"
#include "select_dev.hpp"

namespace lt {

// ---------------------------------------------------------------------------
// Zero the queue counters, the fallback cursor and its chunk counters (a
// kernel, not a memset, so the launch sequence can be captured in a graph).
// ---------------------------------------------------------------------------
__global__ void k_init(uint32_t* qctl) {
  for (int i = threadIdx.x; i < kQctlWords; i += blockDim.x) qctl[i] = 0u;
}

// ---------------------------------------------------------------------------
// Range and initial threshold (sec. 3.2 "Sampling"). One block per row.
// s_min / s_max over the row's visible, finite sample scores; delta = m /
// (s_max - s_min); tau0 = bin of the k-th largest visible sample score, found
// with the sample's histogram. The sample histogram is NOT carried into the
// scan: every sampled key is scanned again, and counting it twice could
// raise the threshold above the true k-th score.
// The sample is the key list `list` (holes < 0 skipped). FROM_SCORES: its
// scores are read from a score matrix (scores-in entry); otherwise from the
// [nq, ns] matrix of sample scores the sample kernel wrote. Each thread keeps
// kRangeUnroll loads in flight: the kernel is bound by load latency.
// ---------------------------------------------------------------------------
constexpr int kRangeThreads = 256;
constexpr int kRangeThreadsLarge = 1024;  // samples of kRangeLargeSample keys or more, or few rows
constexpr int kRangeLargeSample = 16384;
constexpr int kRangeUnroll = 8;

template <int NTH, bool FROM_SCORES>
__device__ __forceinline__ void range_load(const float* rp, const int32_t* list, int ns, RowRange rr, int base,
                                           float (&s)[kRangeUnroll], bool (&vis)[kRangeUnroll]) {
  int key[kRangeUnroll];
#pragma unroll
  for (int u = 0; u < kRangeUnroll; ++u) {
    const int i = base + u * NTH + (int)threadIdx.x;
    key[u] = i < ns ? list[i] : -1;
  }
#pragma unroll
  for (int u = 0; u < kRangeUnroll; ++u) {
    const int i = base + u * NTH + (int)threadIdx.x;
    vis[u] = key[u] >= rr.s && key[u] < rr.e;
    s[u] = vis[u] ? (FROM_SCORES ? rp[key[u]] : rp[i]) : 0.0f;
  }
}

template <int NTH, bool FROM_SCORES>
__global__ __launch_bounds__(NTH) void k_range(const float* src, int64_t stride, int nq, int nk,
                                                         const int32_t* offs, const int32_t* starts,
                                                         const int32_t* list, int ns, int m, int k,
                                                         RowParam* params, int32_t* stats, int32_t* rflag) {
  constexpr int NW = NTH / kWave;
  __shared__ uint32_t hist[kMaxBins];
  __shared__ float red_mn[NW], red_mx[NW];
  __shared__ uint32_t red_n[NW];
  __shared__ uint32_t sel[2];
  const int row = blockIdx.x, wave = threadIdx.x / kWave, l = lane_id();
  const RowRange rr = row_range(offs, starts, row, nk);
  const float* rp = src + (int64_t)row * stride;

  for (int b = threadIdx.x; b < kMaxBins; b += NTH) hist[b] = 0u;
  // the row's flags of the second filter pass (rflag[row]) and of the dense
  // fallback (rflag[nq + row])
  if (rflag && threadIdx.x == 0) {
    rflag[row] = 0;
    rflag[nq + row] = 0;
  }
  float mn = __builtin_inff(), mx = -__builtin_inff();
  uint32_t nvis = 0;
  for (int base = 0; base < ns; base += NTH * kRangeUnroll) {
    float s[kRangeUnroll];
    bool vis[kRangeUnroll];
    range_load<NTH, FROM_SCORES>(rp, list, ns, rr, base, s, vis);
#pragma unroll
    for (int u = 0; u < kRangeUnroll; ++u) {
      nvis += vis[u];
      if (vis[u] && __builtin_isfinite(s[u])) {
        mn = fminf(mn, s[u]);
        mx = fmaxf(mx, s[u]);
      }
    }
  }
  mn = wave_min(mn);
  mx = wave_max(mx);
  nvis = wave_sum(nvis);
  if (l == 0) {
    red_mn[wave] = mn;
    red_mx[wave] = mx;
    red_n[wave] = nvis;
  }
  __syncthreads();
  mn = red_mn[0];
  mx = red_mx[0];
  nvis = red_n[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) {
    mn = fminf(mn, red_mn[w]);
    mx = fmaxf(mx, red_mx[w]);
    nvis += red_n[w];
  }
  float delta = 1.0f, c = 0.0f;
  if (mx > mn) delta = (float)m / (mx - mn);
  if (!(delta > 0.0f) || !__builtin_isfinite(delta)) delta = 1.0f;
  if (__builtin_isfinite(mn)) c = -mn * delta;
  if (!__builtin_isfinite(c)) c = 0.0f;

  for (int base = 0; base < ns; base += NTH * kRangeUnroll) {
    float s[kRangeUnroll];
    bool vis[kRangeUnroll];
    range_load<NTH, FROM_SCORES>(rp, list, ns, rr, base, s, vis);
#pragma unroll
    for (int u = 0; u < kRangeUnroll; ++u) {
      const int b = bin_of(bin_x(s[u], delta, c), m);
      if (vis[u] && b >= 0) atomicAdd(&hist[b], 1u);
    }
  }
  __syncthreads();
  if (wave == 0) {
    const int tau0 = wave_threshold(hist, m, (uint32_t)k, nullptr);
    if (l == 0) params[row] = RowParam{delta, c, tau0, (int)nvis};
    if (stats && l == 0) {
      int32_t* sr = stats + (int64_t)row * LT_ROW_STATS;
      sr[4] = tau0;
      sr[6] = (int32_t)__float_as_uint(delta);
      sr[7] = (int32_t)__float_as_uint(c);
      sr[8] = m;
      sr[9] = (int32_t)nvis;
      sr[10] = 0;
      sr[11] = 0;
    }
  }
  if (!stats) return;
  // The sample's k-th score under the total order (for the invariant
  // kth(sample) <= kth(row) of sec. 3.2 "Sampling"): most-significant-digit
  // radix selection over the order keys of the visible sample scores, four
  // 8-bit digits, the bins reused as the digit histogram.
  uint32_t prefix = 0, pmask = 0, want = (uint32_t)k;
  for (int shift = 24; shift >= 0 && nvis >= (uint32_t)k; shift -= 8) {
    __syncthreads();
    for (int b = threadIdx.x; b < kMaxBins; b += NTH) hist[b] = 0u;
    __syncthreads();
    for (int base = 0; base < ns; base += NTH * kRangeUnroll) {
      float sv[kRangeUnroll];
      bool vis[kRangeUnroll];
      range_load<NTH, FROM_SCORES>(rp, list, ns, rr, base, sv, vis);
#pragma unroll
      for (int u = 0; u < kRangeUnroll; ++u) {
        const uint32_t o = ord_key(sv[u]);
        if (vis[u] && (o & pmask) == prefix) atomicAdd(&hist[(o >> shift) & 0xFFu], 1u);
      }
    }
    __syncthreads();
    if (wave == 0) {
      uint32_t above = 0;
      const int dg = wave_threshold(hist, kMaxBins, want, &above);
      if (l == 0) {
        sel[0] = (uint32_t)dg;
        sel[1] = above;
      }
    }
    __syncthreads();
    const uint32_t dg = sel[0], above = sel[1];
    prefix |= dg << shift;
    pmask |= 0xFFu << shift;
    want -= above;
  }
  if (threadIdx.x == 0)
    stats[(int64_t)row * LT_ROW_STATS + 5] =
        nvis >= (uint32_t)k ? (int32_t)__float_as_uint(ord_inv(prefix)) : (int32_t)0xFF800000u;
}

// ---------------------------------------------------------------------------
// Scores-in filter scan (sec. 3.2 "Filtering" + "Threshold Refresh"). One
// wave owns one (row, key split): it streams its scores once, gates them with
// the row's current threshold bin, appends the passing ones (ballot + mbcnt
// compaction, one write per passing key, key order preserved) to its own
// candidate list and counts them in its own LDS histogram. The threshold is
// kept current after every chunk of 256 keys with the running count of
// candidates above it (see FusedSink in score.hip). A list that reaches `cap`
// stops storing but keeps counting, so the final select can detect the
// overflow.
// ---------------------------------------------------------------------------
constexpr int kFilterWaves = 4;

__global__ __launch_bounds__(kFilterWaves * kWave) void k_filter(
    const float* scores, int64_t stride, int nq, int nk, const int32_t* offs, const int32_t* starts,
    const RowParam* params, int S, int L, int cap, int m, int k, uint32_t* cnt, uint32_t* hist_out, int2* cand) {
  __shared__ uint32_t hist_all[kFilterWaves][kMaxBins];
  const int wave = threadIdx.x / kWave, l = lane_id();
  const int unit = blockIdx.x * kFilterWaves + wave;
  if (unit >= nq * S) return;
  const int row = unit / S, split = unit - row * S;
  uint32_t* hist = hist_all[wave];
  const RowRange rr = row_range(offs, starts, row, nk);
  // the split's keys within the row's range; the first chunk starts on a
  // 4-key boundary for the float4 loads, keys below the range are masked
  const int lo = max(split * L, rr.s & ~3);
  const int hi = min(split * L + L, rr.e);
  const int klo = max(split * L, rr.s);
  const RowParam p = params[row];
  int tau = p.tau0;
  float thr = gate_thr(tau);
  float thr_up = tau < m - 1 ? (float)(tau + 1) : __builtin_nanf("");
  uint32_t above = 0;
  for (int b = l; b < kMaxBins; b += kWave) hist[b] = 0u;
  __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");

  const float* rp = scores + (int64_t)row * stride;
  int2* out = cand + (int64_t)unit * cap;
  uint32_t tail = 0;
  for (int base = lo; base < hi; base += 4 * kWave) {
    const int i0 = base + 4 * l;
    float v[4];
    if (i0 + 3 < hi) {
      float4 t = *reinterpret_cast<const float4*>(rp + i0);
      v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) v[j] = (i0 + j < hi) ? rp[i0 + j] : 0.0f;
    }
    float x[4];
    bool ps[4];
    uint32_t below = 0, total = 0, up = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[j] = bin_x(v[j], p.delta, p.c);
      ps[j] = (i0 + j >= klo) && (i0 + j < hi) && !(x[j] < thr);
      uint64_t mask = __ballot(ps[j]);
      below += mbcnt64(mask);
      total += (uint32_t)__popcll(mask);
      up += (uint32_t)__popcll(__ballot(ps[j] && x[j] >= thr_up));
    }
    if (total == 0) continue;  // wave-uniform
    uint32_t pos = tail + below;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (ps[j]) {
        if (pos < (uint32_t)cap) out[pos] = make_int2(i0 + j, __float_as_int(v[j]));
        int b = bin_of(x[j], m);
        if (b >= 0) atomicAdd(&hist[b], 1u);
        ++pos;
      }
    }
    tail += total;
    above += up;
    if (above >= (uint32_t)k) {
      __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
      while (above >= (uint32_t)k && tau < m - 1) {
        ++tau;
        above -= hist[tau];
      }
      thr = gate_thr(tau);
      thr_up = tau < m - 1 ? (float)(tau + 1) : __builtin_nanf("");
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  for (int b = l; b < m; b += kWave) hist_out[(int64_t)unit * m + b] = hist[b];
  if (l == 0) cnt[unit] = tail;
}

// ---------------------------------------------------------------------------
// Final select (sec. 3.2 "Top-k Selection"). One block per row.
//  1. Sum the row's HS histograms; the final threshold bin tau is the largest
//     bin whose suffix count reaches k (bins >= tau are complete: every key in
//     them passed the gate, which never exceeded tau).
//  2. Candidates in bins above tau (fewer than k) go straight to the output,
//     in list order.
//  3. Candidates in bin tau are collected in LDS and only they are sorted;
//     the best k - (count above) complete the row.
// The row's S lists are walked as one sequence, NTH lists at a time (their
// counts prefix-summed in LDS) and PER entries per thread per step, so many
// short lists cost no more than one long one. Keyed rows (few rows with
// hundreds of thousands of candidates each) run 1024 threads with 8 entries
// per thread; the others 256 threads with 4.
// Rows whose buffer overflowed, whose threshold bin does not fit in LDS,
// whose counts disagree with their lists, whose final bin lies below the
// sample's initial bin, or that are forced, are queued for the exact fallback
// instead.
// ---------------------------------------------------------------------------
constexpr int kSelThreads = 256;
constexpr int kSelPer = 4;         // list entries per thread per step
constexpr int kSelThreadsWide = 1024;  // keyed rows, and launches of few rows
constexpr int kSelPerWide = 8;
constexpr int kSelFewRows = 512;     // launches of at most this many rows use the wide blocks
constexpr int kSecondSelectGrid = 512;  // blocks of the second select (persistent over its queue)

// Threshold bins of at most this many keys are ranked by counting instead of
// sorted.
constexpr int kRankMax = 512;

// LDS byte offset of the sort entries of k_select with NTH threads.
constexpr size_t select_ent_offset(int nth) { return ((size_t)kMaxBins + 32 + nth + 16) * 4; }

template <int NTH, int PER>
__device__ __forceinline__ void select_row(int row, RowParam* params, const uint32_t* cnt, const uint32_t* hist,
                           const int2* cand, int nq, int S, int HS, int cap, int m, int k, int E, uint32_t flags,
                           int32_t* out_i, float* out_s, uint32_t* qctl, int32_t* queue, int32_t* rqueue,
                           int32_t* rflag, int32_t* stats) {
  extern __shared__ __align__(16) uint8_t lds[];
  uint32_t* hsum = reinterpret_cast<uint32_t*>(lds);          // [256]
  uint32_t* tmp = hsum + kMaxBins;                             // [32]
  uint32_t* off = tmp + 32;                                    // [NTH + 1]: list offsets of a group
  uint64_t* ent = reinterpret_cast<uint64_t*>(lds + select_ent_offset(NTH));  // [E]
  const int tid = threadIdx.x;
  // keyed: the lists are not in key order, so the tie-break position is the
  // key itself, the sorted scores are rebuilt from the sort entries, and
  // every row is sorted (the order of arrival would make it vary between
  // calls)
  const bool keyed = flags & kSelKeyed;
  const bool ilv = flags & kSelIlv;
  const bool sorted = (flags & LT_SORTED_OUTPUT) || keyed;
  int32_t* oi = out_i + (int64_t)row * k;
  float* os = out_s + (int64_t)row * k;

  // ---- overflow / forced ----
  uint32_t total_c = 0;
  int reason = (flags & LT_FORCE_FALLBACK) ? 3 : 0;
  {
    uint32_t my = 0;
    bool ovf = false;
    for (int s = tid; s < S; s += NTH) {
      const uint32_t c = cnt[(int64_t)row * S + s];
      my += c;
      ovf |= c > (uint32_t)cap;
    }
    (void)block_scan_excl<NTH>(my, tmp, &total_c);
    if (__syncthreads_or(ovf) && reason == 0) reason = 1;
  }
  auto enqueue = [&](int why, int tau, uint32_t nt) {
    if (tid == 0) {
      uint32_t slot = atomicAdd(&qctl[0], 1u);
      queue[slot] = row;
      if (rflag) rflag[nq + row] = 1;  // queued for the dense fallback
      if (stats) {
        int32_t* st = stats + (int64_t)row * LT_ROW_STATS;
        if (!(flags & kSelSecond)) st[0] = (int32_t)total_c;
        st[1] = tau;
        st[2] = why;
        st[3] = (int32_t)nt;
      }
    }
  };
  if (reason == 3) {
    enqueue(reason, -2, 0);
    return;
  }

  // ---- 1. final threshold bin ----
  for (int b = tid; b < kMaxBins; b += NTH) {
    uint32_t h = 0;
    if (b < m)
      for (int s = 0; s < HS; ++s) h += hist[((int64_t)row * HS + s) * m + b];
    hsum[b] = h;
  }
  __syncthreads();
  if (tid < kWave) {
    uint32_t above = 0;
    int tau = wave_threshold(hsum, m, (uint32_t)k, &above);
    if (tid == 0) {
      tmp[24] = (uint32_t)tau;
      tmp[25] = above;
    }
  }
  __syncthreads();
  const int tau = (int)tmp[24];
  const uint32_t c_above = tmp[25];
  const uint32_t c_tie = tau >= 0 ? hsum[tau] : 0u;
  __syncthreads();
  if (reason == 1) {
    // The lists overflowed, but the histograms kept counting: bins >= tau
    // are complete and tau is the row's exact final bin. A second filter
    // pass gated at tau from its first key writes exactly the c_above +
    // c_tie keys of those bins; when they fit in one list (and the sort
    // buffer) the row is queued for that pass, else for the dense fallback.
    if ((flags & kSelRefilter) && tau >= 0 && c_above + c_tie <= (uint32_t)cap && c_tie <= (uint32_t)E) {
      if (tid == 0) {
        params[row].tau0 = tau;
        rflag[row] = 1;
        rqueue[atomicAdd(&qctl[1], 1u)] = row;
        if (stats) {
          int32_t* st = stats + (int64_t)row * LT_ROW_STATS;
          st[0] = (int32_t)total_c;
          st[1] = tau;
          st[2] = 6;
          st[3] = (int32_t)c_tie;
        }
      }
      return;
    }
    enqueue(1, tau, c_tie);
    return;
  }
  const RowParam p = params[row];
  // Every visible sample key in a bin >= tau0 passes the gate or is
  // outranked by k counted keys, so an exact scan ends with tau >= tau0. A
  // lower bin means the sample's scores and the scan's disagree; the bins
  // between were gated and are incomplete, so the row is recomputed.
  if (p.tau0 >= 0 && tau < p.tau0) {
    enqueue(5, tau, 0);
    return;
  }

  // ---- 2./3. one pass over the candidates ----
  uint32_t run_above = 0, run_tie = 0;
  bool tie_ovf = false;
  if (keyed) {
    // The final sort puts the keys above bin tau in order and bin tau's
    // entries carry their keys, so no position needs the list order: each
    // wave takes whole lists, four at a time when there are enough (16 lanes
    // on 16 consecutive positions of each, one 128-byte chunk), with PER
    // loads in flight per lane, and reserves output slots with one LDS
    // atomic per kind and step. No block-wide step, no search for a
    // position's list.
    constexpr int NW = NTH / kWave;
    const int wave = tid / kWave, l = lane_id();
    const int lpw = S >= 4 * NW ? 4 : 1;  // lists a wave takes at once
    const int ll = kWave / lpw, sub = l / ll, lo = l - sub * ll;
    if (tid == 0) {
      tmp[26] = 0u;
      tmp[27] = 0u;
    }
    __syncthreads();
    for (int s0 = wave * lpw; s0 < S; s0 += NW * lpw) {
      const int s = s0 + sub;
      const int64_t li = (int64_t)row * S + s;
      const uint32_t c = s < S ? min(cnt[li], (uint32_t)cap) : 0u;
      // the wave steps through the longest of its lists
      uint32_t cmax = 0u;
      for (int g = 0; g < lpw; ++g) cmax = max(cmax, (uint32_t)__builtin_amdgcn_readlane((int)c, g * ll));
      for (uint32_t p0 = 0; p0 < cmax; p0 += (uint32_t)(PER * ll)) {
        int2 ce[PER];
#pragma unroll
        for (int u = 0; u < PER; ++u) {
          const uint32_t pos = p0 + (uint32_t)(u * ll + lo);
          ce[u] = make_int2(0, 0);
          if (pos < c) ce[u] = cand[ilv ? ilv_index(li, pos, (int64_t)nq * S) : li * cap + pos];
        }
        // bit u: entry u is above bin tau (ab) / in it (ti); the wave masks
        // are taken again where they are used, to keep few of them live
        uint32_t ab = 0u, ti = 0u, na = 0u, nt = 0u;
#pragma unroll
        for (int u = 0; u < PER; ++u) {
          const bool v = p0 + (uint32_t)(u * ll + lo) < c;
          const int b = bin_of(bin_x(__int_as_float(ce[u].y), p.delta, p.c), m);
          const bool a1 = v & (b > tau), t1 = v & (b == tau);
          ab |= (uint32_t)a1 << u;
          ti |= (uint32_t)t1 << u;
          na += (uint32_t)__popcll(__ballot(a1));
          nt += (uint32_t)__popcll(__ballot(t1));
        }
        uint32_t ba = 0u, bt = 0u;
        if (l == 0) {
          if (na) ba = atomicAdd(&tmp[26], na);
          if (nt) bt = atomicAdd(&tmp[27], nt);
        }
        ba = (uint32_t)__builtin_amdgcn_readfirstlane((int)ba);
        bt = (uint32_t)__builtin_amdgcn_readfirstlane((int)bt);
#pragma unroll
        for (int u = 0; u < PER; ++u) {
          const bool a1 = (ab >> u) & 1u, t1 = (ti >> u) & 1u;
          const uint64_t ma = __ballot(a1), mt = __ballot(t1);
          if (a1) {
            const uint32_t r = ba + mbcnt64(ma);
            if (r < (uint32_t)k) {
              oi[r] = ce[u].x;
              os[r] = __int_as_float(ce[u].y);
            }
          }
          if (t1) {
            const uint32_t r = bt + mbcnt64(mt);
            if (r < (uint32_t)E) ent[r] = comp_key(__int_as_float(ce[u].y), (uint32_t)ce[u].x);
          }
          ba += (uint32_t)__popcll(ma);
          bt += (uint32_t)__popcll(mt);
        }
      }
    }
    __syncthreads();
    run_above = tmp[26];
    run_tie = tmp[27];
  }
  // lists in key order: one block-wide pass in list order, so that a
  // position in the concatenated lists orders equal scores by key
  for (int g0 = 0; g0 < (keyed ? 0 : S); g0 += NTH) {
    // offsets of the group's lists in their concatenation
    const int sg = g0 + tid;
    const uint32_t cg = sg < S ? min(cnt[(int64_t)row * S + sg], (uint32_t)cap) : 0u;
    uint32_t gtot;
    const uint32_t ex = block_scan_excl<NTH>(cg, tmp, &gtot);
    off[tid] = ex;
    if (tid == 0) off[NTH] = gtot;
    __syncthreads();
    const int ng = min(NTH, S - g0);
    for (uint32_t base = 0; base < gtot; base += NTH * PER) {
      int2 ce[PER];
      uint32_t gpos[PER];
      bool ab[PER], ti[PER];
      uint32_t na = 0, nt = 0;
      // the PER positions of a thread are consecutive: one binary search for
      // the list holding the first (the last list whose offset is <= i), a
      // forward walk for the others; then every load goes out before any is
      // used, so a step costs one load latency, not PER of them
      const uint32_t i0 = base + (uint32_t)(tid * PER);
      int lst[PER];
      {
        int lo = 0, hi = ng - 1;
        const uint32_t i = i0 < gtot ? i0 : gtot - 1;
        while (lo < hi) {
          const int mid = (lo + hi + 1) >> 1;
          if (off[mid] <= i) lo = mid;
          else hi = mid - 1;
        }
#pragma unroll
        for (int j = 0; j < PER; ++j) {
          while (lo + 1 < ng && off[lo + 1] <= i0 + (uint32_t)j) ++lo;
          lst[j] = lo;
        }
      }
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const uint32_t i = i0 + (uint32_t)j;
        ce[j] = make_int2(0, 0);
        if (i < gtot) {
          const int64_t li = (int64_t)row * S + g0 + lst[j];
          const uint32_t pos = i - off[lst[j]];
          ce[j] = cand[ilv ? ilv_index(li, pos, (int64_t)nq * S) : li * cap + pos];
        }
      }
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const uint32_t i = i0 + (uint32_t)j;
        ab[j] = ti[j] = false;
        gpos[j] = 0;
        if (i < gtot) {
          // the list position, which increases with the key index
          gpos[j] = (uint32_t)(g0 + lst[j]) * (uint32_t)cap + (i - off[lst[j]]);
          const int b = bin_of(bin_x(__int_as_float(ce[j].y), p.delta, p.c), m);
          ab[j] = b > tau;
          ti[j] = b == tau;
        }
        na += ab[j];
        nt += ti[j];
      }
      uint32_t tot;
      const uint32_t ex2 = block_scan_excl<NTH>((na << 16) | nt, tmp, &tot);
      uint32_t ra = run_above + (ex2 >> 16), rt = run_tie + (ex2 & 0xFFFFu);
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        if (ab[j] && ra < (uint32_t)k) {
          oi[ra] = ce[j].x;
          os[ra] = __int_as_float(ce[j].y);
        }
        if (ti[j] && rt < (uint32_t)E) ent[rt] = comp_key(__int_as_float(ce[j].y), gpos[j]);
        ra += ab[j];
        rt += ti[j];
      }
      run_above += tot >> 16;
      run_tie += tot & 0xFFFFu;
    }
    __syncthreads();  // off[] is rewritten by the next group
  }
  const uint32_t nent = run_tie;
  tie_ovf = nent > (uint32_t)E;
  if (tie_ovf || run_above != c_above) {
    enqueue(tie_ovf ? 2 : 4, tau, run_tie);
    return;
  }
  // the need = k - c_above best keys of bin tau, after the keys above it
  const uint32_t need = (uint32_t)k - c_above;
  const uint32_t take = min(need, nent);
  // the bin's i-th best key goes to slot c_above + i
  auto emit = [&](uint32_t i, uint64_t e) {
    const uint32_t gp = comp_pos(e);
    if (keyed) {
      oi[c_above + i] = (int32_t)gp;
      os[c_above + i] = ord_inv((uint32_t)(e >> 32));
      return;
    }
    const uint32_t s = gp / (uint32_t)cap, j = gp - s * (uint32_t)cap;
    const int2 ce = cand[((int64_t)row * S + s) * cap + j];
    oi[c_above + i] = ce.x;
    os[c_above + i] = __int_as_float(ce.y);
  };
  if (nent <= (uint32_t)kRankMax) {
    // a small bin: each key's rank is the number of keys above it (the sort
    // entries are distinct), one pass over the bin per key and no barrier
    // per sorting stage
    __syncthreads();
    for (uint32_t i = tid; i < nent; i += NTH) {
      const uint64_t e = ent[i];
      uint32_t r = 0;
      for (uint32_t j = 0; j < nent; ++j) r += ent[j] > e;
      if (r < take) emit(r, e);
    }
  } else {
    const int P = next_pow2((int)nent);
    for (int i = tid; i < P; i += NTH)
      if ((uint32_t)i >= nent) ent[i] = 0ull;
    __syncthreads();
    bitonic_sort_desc_fast<NTH>(ent, P);
    for (uint32_t i = tid; i < take; i += NTH) emit(i, ent[i]);
  }
  for (uint32_t i = c_above + take + tid; i < (uint32_t)k; i += NTH) {
    oi[i] = -1;
    os[i] = -__builtin_inff();
  }
  if (sorted) {
    // Sort the row's nout kept keys in place. Equal scores lie in one bin, and
    // within a bin the row already holds them in key order (the list order,
    // or the bin's sort), so (score, slot) is the total order; keyed rows,
    // whose keys above bin tau came in arrival order, sort by (score, key)
    // and take canonical scores from the sort entries. The slots' pairs wait
    // in the upper half of the sort buffer (k <= E / 2).
    const uint32_t nout = c_above + take;
    int2* pair = reinterpret_cast<int2*>(ent + E / 2);
    __threadfence_block();
    __syncthreads();
    for (uint32_t i = tid; i < nout; i += NTH) {
      const int32_t x = oi[i];
      const float y = os[i];
      pair[i] = make_int2(x, __float_as_int(y));
      ent[i] = comp_key(y, keyed ? (uint32_t)x : i);
    }
    const int P = next_pow2((int)nout < 1 ? 1 : (int)nout);
    for (int i = tid; i < P; i += NTH)
      if ((uint32_t)i >= nout) ent[i] = 0ull;
    __syncthreads();
    bitonic_sort_desc_fast<NTH>(ent, P);
    for (uint32_t i = tid; i < nout; i += NTH) {
      const uint32_t g = comp_pos(ent[i]);
      if (keyed) {
        oi[i] = (int32_t)g;
        os[i] = ord_inv((uint32_t)(ent[i] >> 32));
      } else {
        const int2 pr = pair[g];
        oi[i] = pr.x;
        os[i] = __int_as_float(pr.y);
      }
    }
  }
  if (stats && tid == 0) {
    int32_t* st = stats + (int64_t)row * LT_ROW_STATS;
    // a row finished by the second filter pass keeps its candidates written
    // by the first pass (field 0) and reports reason 6
    if (!(flags & kSelSecond)) st[0] = (int32_t)total_c;
    st[1] = tau;
    st[2] = (flags & kSelSecond) ? 6 : 0;
    st[3] = (int32_t)run_tie;
  }
}

// One block per row.
template <int NTH, int PER>
__global__ __launch_bounds__(NTH) void k_select(
    RowParam* params, const uint32_t* cnt, const uint32_t* hist, const int2* cand, int nq,
    int S, int HS, int cap, int m, int k, int E, uint32_t flags, int32_t* out_i, float* out_s,
    uint32_t* qctl, int32_t* queue, int32_t* rqueue, int32_t* rflag, int32_t* stats) {
  select_row<NTH, PER>(blockIdx.x, params, cnt, hist, cand, nq, S, HS, cap, m, k, E, flags, out_i, out_s, qctl,
                       queue, rqueue, rflag, stats);
}

// The rows of the second filter pass (queue rqueue, length qctl[1]);
// persistent: block b takes entries b, b + grid, ...
template <int NTH, int PER>
__global__ __launch_bounds__(NTH) void k_select_second(
    RowParam* params, const uint32_t* cnt, const uint32_t* hist, const int2* cand, int nq,
    int S, int HS, int cap, int m, int k, int E, uint32_t flags, int32_t* out_i, float* out_s,
    uint32_t* qctl, int32_t* queue, int32_t* rqueue, int32_t* rflag, int32_t* stats) {
  const uint32_t n = qctl[1];
  for (uint32_t i = blockIdx.x; i < n; i += gridDim.x) {
    select_row<NTH, PER>(rqueue[i], params, cnt, hist, cand, nq, S, HS, cap, m, k, E, flags | kSelSecond, out_i,
                         out_s, qctl, queue, rqueue, rflag, stats);
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Exact fallback for the scores-in entry: the queued rows go through plain
// radix selection over all their visible scores. Persistent: block b handles
// queue entries b, b + grid, ...; the queue length is read on the device.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kSelThreads) void k_fallback_scores(
    const float* scores, int64_t stride, int nk, const int32_t* offs, const int32_t* starts, int k,
    uint32_t flags, uint32_t* qctl, const int32_t* queue, int32_t* cidx, float* cscore, int32_t* out_i,
    float* out_s) {
  extern __shared__ __align__(16) uint8_t lds[];
  __shared__ int last;
  const uint32_t n = qctl[0];
  // split mode (few rows: up to kFallbackGrid blocks over the rows' chunks,
  // no scratch rows needed), else one block per queued row
  const int chunks = fallback_chunks(n, min((int)gridDim.x, kFallbackGrid), INT_MAX, nk);
  if (chunks > 1) {
    if (blockIdx.x >= n * (uint32_t)chunks) return;  // block-uniform
    const int e = blockIdx.x / chunks, c = blockIdx.x - e * chunks;
    const int row = queue[e];
    const RowRange rr = row_range(offs, starts, row, nk);
    const int len = rr.e > rr.s ? rr.e - rr.s : 0, per = (len + chunks - 1) / chunks;
    const int kb = min(rr.s + c * per, rr.s + len), ke = min(kb + per, rr.s + len);
    const int64_t cb = (int64_t)e * chunks * k;
    split_fallback_select<kSelThreads>(scores + (int64_t)row * stride, rr.s, len, per, chunks, c, kb, ke, k,
                                       cidx + cb, cscore + cb, &qctl[kQctlDone + e], out_i + (int64_t)row * k,
                                       out_s + (int64_t)row * k, flags & LT_SORTED_OUTPUT, lds, &last);
    return;
  }
  for (uint32_t r = blockIdx.x; r < n; r += gridDim.x) {
    const int row = queue[r];
    const RowRange rr = row_range(offs, starts, row, nk);
    radix_select_row<kSelThreads>(scores + (int64_t)row * stride + rr.s, rr.e - rr.s, k,
                                  out_i + (int64_t)row * k, out_s + (int64_t)row * k,
                                  flags & LT_SORTED_OUTPUT, lds, rr.s);
    __syncthreads();
  }
}

// Plain radix selection of every row (no sampling, no filtering).
__global__ __launch_bounds__(kSelThreads) void k_radix(const float* scores, int64_t stride, int nk,
                                                       const int32_t* offs, int k, uint32_t flags,
                                                       int32_t* out_i, float* out_s) {
  extern __shared__ __align__(16) uint8_t lds[];
  const int row = blockIdx.x;
  int e = offs ? offs[row] : nk;
  e = e < 0 ? 0 : (e > nk ? nk : e);
  radix_select_row<kSelThreads>(scores + (int64_t)row * stride, e, k, out_i + (int64_t)row * k,
                                out_s + (int64_t)row * k, flags & LT_SORTED_OUTPUT, lds);
}

// The fused path's dense fallback mode, second half: queued row t (flag 1)
// was re-scored into scratch row t; one block selects it.
__global__ __launch_bounds__(kSelThreads) void k_fallback_rows(const uint32_t* qctl, const int32_t* fbflag,
                                                               const float* scratch, int nq, int nk,
                                                               const int32_t* offs, const int32_t* starts, int k,
                                                               uint32_t flags, int slots, int qt, int32_t* out_i,
                                                               float* out_s) {
  extern __shared__ __align__(16) uint8_t lds[];
  const int row = blockIdx.x;
  if (!fallback_dense(qctl[0], nq, kFallbackGrid, slots, nk, qt) || fbflag[row] != 1) return;  // block-uniform
  const RowRange rr = row_range(offs, starts, row, nk);
  radix_select_row<kSelThreads>(scratch + (int64_t)row * nk + rr.s, rr.e - rr.s, k, out_i + (int64_t)row * k,
                                out_s + (int64_t)row * k, flags & LT_SORTED_OUTPUT, lds, rr.s);
}

// ---------------------------------------------------------------------------
// Host launchers
// ---------------------------------------------------------------------------
hipError_t launch_init(uint32_t* qctl, hipStream_t st) {
  hipLaunchKernelGGL(k_init, dim3(1), dim3(64), 0, st, qctl);
  return hipGetLastError();
}

hipError_t launch_range(bool from_scores, const float* src, int64_t stride, int nq, int nk,
                        const int32_t* offs, const int32_t* starts, const int32_t* list, int ns, int m, int k,
                        RowParam* params, int32_t* stats, int32_t* rflag, hipStream_t st) {
  dim3 grid(nq);
  auto go = [&](auto kernel, int nth) {
    hipLaunchKernelGGL(kernel, grid, dim3(nth), 0, st, src, stride, nq, nk, offs, starts, list, ns, m, k, params,
                       stats, rflag);
  };
  // a long sample is read in fewer, wider steps (the kernel waits on loads);
  // so are the rows of a launch of few rows, which otherwise leaves most of
  // the GPU idle
  const bool large = ns >= kRangeLargeSample || nq <= kSelFewRows;
  if (from_scores) {
    if (large) go(k_range<kRangeThreadsLarge, true>, kRangeThreadsLarge);
    else go(k_range<kRangeThreads, true>, kRangeThreads);
  } else {
    if (large) go(k_range<kRangeThreadsLarge, false>, kRangeThreadsLarge);
    else go(k_range<kRangeThreads, false>, kRangeThreads);
  }
  return hipGetLastError();
}

hipError_t launch_filter(const float* scores, int64_t stride, int nq, int nk, const int32_t* offs,
                         const int32_t* starts, const RowParam* params, int S, int L, int cap, int m, int k,
                         uint32_t* cnt, uint32_t* hist, int2* cand, hipStream_t st) {
  const int units = nq * S;
  dim3 grid((units + kFilterWaves - 1) / kFilterWaves);
  hipLaunchKernelGGL(k_filter, grid, dim3(kFilterWaves * kWave), 0, st, scores, stride, nq, nk, offs, starts,
                     params, S, L, cap, m, k, cnt, hist, cand);
  return hipGetLastError();
}

size_t select_lds_bytes(int E) { return select_ent_offset(kSelThreadsWide) + (size_t)E * 8; }

hipError_t launch_select(RowParam* params, const uint32_t* cnt, const uint32_t* hist, const int2* cand, int nq,
                         int S, int HS, int cap, int m, int k, int E, uint32_t flags, int32_t* out_i, float* out_s,
                         uint32_t* qctl, int32_t* queue, int32_t* rqueue, int32_t* rflag, int32_t* stats,
                         hipStream_t st) {
  auto go = [&](auto kernel, int nth) {
    const size_t lds = select_ent_offset(nth) + (size_t)E * 8;
    if (lds > 65536) (void)hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(kernel, dim3(nq), dim3(nth), lds, st, params, cnt, hist, cand, nq, S, HS, cap, m, k, E, flags,
                       out_i, out_s, qctl, queue, rqueue, rflag, stats);
  };
  // one block per row: a launch of few rows (a short chunk) fills the GPU
  // only with wide blocks, whose more loads in flight also shorten the walk
  // over the lists; many rows fill it with narrow ones (measured on MI355X:
  // 256 rows, 33 K candidates each, 1.57 -> 0.79 ms; 4096 rows with 8.7 K,
  // 0.16 ms at 256 threads against 0.37 ms at 1024)
  if ((flags & kSelIlv) || nq <= kSelFewRows) go(k_select<kSelThreadsWide, kSelPerWide>, kSelThreadsWide);
  else go(k_select<kSelThreads, kSelPer>, kSelThreads);
  return hipGetLastError();
}

hipError_t launch_select_second(RowParam* params, const uint32_t* cnt, const uint32_t* hist, const int2* cand,
                                int nq, int S, int HS, int cap, int m, int k, int E, uint32_t flags, int32_t* out_i,
                                float* out_s, uint32_t* qctl, int32_t* queue, int32_t* rqueue, int32_t* rflag,
                                int32_t* stats,
                                hipStream_t st) {
  const int grid = nq < kSecondSelectGrid ? nq : kSecondSelectGrid;
  if (grid == 0) return hipSuccess;
  auto go = [&](auto kernel, int nth) {
    const size_t lds = select_ent_offset(nth) + (size_t)E * 8;
    if (lds > 65536) (void)hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(kernel, dim3(grid), dim3(nth), lds, st, params, cnt, hist, cand, nq, S, HS, cap, m, k, E,
                       flags & ~kSelRefilter, out_i, out_s, qctl, queue, rqueue, rflag, stats);
  };
  if (flags & kSelIlv) go(k_select_second<kSelThreadsWide, kSelPerWide>, kSelThreadsWide);
  else go(k_select_second<kSelThreads, kSelPer>, kSelThreads);
  return hipGetLastError();
}

hipError_t launch_fallback_scores(const float* scores, int64_t stride, int nk, const int32_t* offs,
                                  const int32_t* starts, int k, uint32_t flags, uint32_t* qctl,
                                  const int32_t* queue, int32_t* cidx, float* cscore, int32_t* out_i, float* out_s,
                                  int grid, hipStream_t st) {
  if (radix_lds_bytes(k) > 65536)
    (void)hipFuncSetAttribute((const void*)k_fallback_scores, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)radix_lds_bytes(k));
  hipLaunchKernelGGL(k_fallback_scores, dim3(grid), dim3(kSelThreads), radix_lds_bytes(k), st, scores,
                     stride, nk, offs, starts, k, flags, qctl, queue, cidx, cscore, out_i, out_s);
  return hipGetLastError();
}

hipError_t launch_fallback_rows(const uint32_t* qctl, const int32_t* fbflag, const float* scratch, int nq, int nk,
                                const int32_t* offs, const int32_t* starts, int k, uint32_t flags, int slots,
                                int qt, int32_t* out_i, float* out_s, hipStream_t st) {
  if (nq <= 0 || nq > slots || qt > 64) return hipSuccess;  // the dense mode cannot hold
  const size_t lds = radix_lds_bytes(k);
  if (lds > 65536)
    (void)hipFuncSetAttribute((const void*)k_fallback_rows, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  hipLaunchKernelGGL(k_fallback_rows, dim3(nq), dim3(kSelThreads), lds, st, qctl, fbflag, scratch, nq, nk, offs,
                     starts, k, flags, slots, qt, out_i, out_s);
  return hipGetLastError();
}

hipError_t launch_radix(const float* scores, int64_t stride, int nq, int nk, const int32_t* offs,
                        int k, uint32_t flags, int32_t* out_i, float* out_s, hipStream_t st) {
  if (radix_lds_bytes(k) > 65536)
    (void)hipFuncSetAttribute((const void*)k_radix, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)radix_lds_bytes(k));
  hipLaunchKernelGGL(k_radix, dim3(nq), dim3(kSelThreads), radix_lds_bytes(k), st, scores, stride, nk,
                     offs, k, flags, out_i, out_s);
  return hipGetLastError();
}

}  // namespace lt
