// Wide-vector scan for the paper's retrieval shapes (sec. 4.1 "Large-Scale
// Retrieval Benchmark": 768-dimensional passage embeddings, batches of 64
// queries, corpora of millions of items, k up to 8192).
//
// The 128-dimensional scorer keeps each wave's queries stationary in VGPRs;
// at 768 dimensions 32 queries alone would take 192 VGPRs. This scan turns
// the layout around:
//  * a block owns 64 queries, held in LDS as ready-made MFMA A fragments
//    (2 M tiles x D/16 K steps x 1 KB, read conflict-free, one 16-byte read
//    per lane per fragment);
//  * each wave streams its own tiles of 32 items straight from HBM into B
//    fragments (no LDS staging), keeping PD fragments in flight in a register
//    ring that runs across tile boundaries;
//  * a wave tile is the whole 64 x 32 score block, so each item is read from
//    HBM once per block and the waves of a block need no barrier in the scan.
// 64 queries make 64 flops per item byte, a fifth of the bf16 MFMA ridge
// point: the scan is bound by HBM, and the design goal is bytes in flight.
//
// Fused filter (sec. 3.2 "Filtering", "Threshold Refresh"). A 64-query batch
// needs about 256 key splits to fill the GPU, and a threshold refreshed from
// one split's own histogram can only reach that split's local top-k, which
// for large k admits most of the split. Here all splits of a row share one
// histogram and one threshold bin in global memory (the paper's per-CTA
// structure widened to the grid), while each block keeps its own candidate
// list per row:
//  * a tile's passing candidates reserve their slots in the block's list with
//    one LDS atomic add per query and count themselves in the block's LDS
//    histogram of the row;
//  * wave w of a block looks after rows w, w + 8, ..., one per tile in turn:
//    it moves the block's LDS counts of the row into the row's shared
//    histogram (one atomic add per non-empty bin), reads the shared
//    histogram and the row's published bin, and one tile later walks the
//    histogram from the top for the threshold bin, raises the block's bin in
//    LDS and, when it beats the published one, publishes it with an atomic
//    max; every wave takes the block's bins from LDS once per tile.
// (Device-wide atomics and coherent reads per query and tile, or per
// candidate, contended by 2048 waves for 64 rows, cost more than the scan.)
// A published bin b had, when it was computed, at least k counted candidates
// in bins >= b. Counts only grow, so b never exceeds the final threshold bin
// the select stage computes, and every key a gate drops lies below it. A
// stale bin only loosens the gate.
#include <utility>

#include "internal.hpp"
#include "select_dev.hpp"

namespace lt {

typedef __bf16 wbf16x8_t __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) uint32_t lds_u32_t;
typedef __attribute__((address_space(3))) int lds_i32_t;
typedef uint32_t wu32x4_t __attribute__((ext_vector_type(4)));

// Cache policy of a device-coherent load (sc1, as for agent-scope atomics).
constexpr int kCoherent = 0x10;
typedef float wf32x16_t __attribute__((ext_vector_type(16)));
typedef int wi32x4_t __attribute__((ext_vector_type(4)));

template <int N, class F>
__device__ __forceinline__ void wstatic_for(F&& f) {
  [&]<int... I>(std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
  }(std::make_integer_sequence<int, N>{});
}

template <int D_, bool RELU_>
struct WCfg {
  static constexpr int D = D_;
  static constexpr bool RELU = RELU_;
  static constexpr int KS = D / 16;          // bf16 32x32x16 K steps per item
  static constexpr int ROWB = D * 2;         // bytes per item row
  static constexpr int MT = 2;               // M tiles of 32 queries
  static constexpr int QT = 32 * MT;         // queries per block
  static constexpr int WAVES = 8;
  static constexpr int NTHREADS = WAVES * kWave;
  static constexpr int KT = 32;              // items per wave tile
  static constexpr int STEP = KT * WAVES;    // items per block step
  static constexpr int PD = 16;              // B fragments in flight per wave (16 KB)
  static constexpr int LG = 4;               // B loads per 128-byte line of a row, issued together
  static constexpr int NI = 16 * MT;         // scores per lane per tile
  static constexpr int REFRESH = 8;          // tiles between two refreshes of one wave
  static constexpr int Q_LDS = MT * KS * kWave * 16;
  static_assert(D % 16 == 0 && KS % PD == 0, "the fragment ring must divide the K steps");
  static_assert(PD % LG == 0 && KS % LG == 0, "load groups must tile the ring and the K steps");
  static_assert(NI == 32, "one bit per score item");
};

// Query (within the block) of score item it = 16 * mt + v, accumulator
// register v of M tile mt, in lane half h: row 8 * (v / 4) + 4 * h + v % 4 of
// the M tile. Each query is exactly one (item, half) pair.
__host__ __device__ constexpr int wq_of(int it, int h) {
  return 32 * (it >> 4) + 8 * ((it & 15) >> 2) + 4 * h + (it & 3);
}

// Queries q0 .. q0 + 63 into LDS as A fragments: fragment (mt, ks) is 1 KB at
// ((mt * KS + ks) * 64) * 16, lane l's 16 bytes are elements
// [16 ks + 8 (l / 32), +8) of query 32 mt + l % 32 (zero past the last query).
template <class C>
__device__ __forceinline__ void wide_load_q(uint8_t* qlds, const ScoreArgs& a, int q0) {
  const uint16_t* q = static_cast<const uint16_t*>(a.q);
  for (int u = threadIdx.x; u < C::MT * C::KS * kWave; u += C::NTHREADS) {
    const int f = u / kWave, l = u % kWave, mt = f / C::KS, ks = f % C::KS;
    const int t = q0 + 32 * mt + (l & 31);
    wi32x4_t v = {0, 0, 0, 0};
    if (t < a.nq) v = *reinterpret_cast<const wi32x4_t*>(q + (int64_t)t * C::D + 16 * ks + 8 * (l >> 5));
    *reinterpret_cast<wi32x4_t*>(qlds + (size_t)u * 16) = v;
  }
  __syncthreads();
}

// Weight of the query of each score item (1 without weights, 0 past the end).
template <class C>
__device__ __forceinline__ void wide_weights(float (&wv)[C::NI], const ScoreArgs& a, int q0) {
  const int h = lane_id() >> 5;
#pragma unroll
  for (int it = 0; it < C::NI; ++it) {
    const int t = q0 + wq_of(it, h);
    wv[it] = t < a.nq ? (a.w ? a.w[t] : 1.0f) : 0.0f;
  }
}

struct WSrcContig {
  __device__ int key(int i) const { return i; }
};
struct WSrcList {
  const int32_t* list;
  __device__ int key(int i) const {
    const int v = list[i];
    return v < 0 ? 0 : v;
  }
};

// One wave's share of the scan over positions [kbeg, kend) of `src`: tiles
// wave, wave + WAVES, ... of 32 positions. Lane (r32, h) reads item
// kbeg + 32 t + r32 (clamped to the last position; consumers mask it) and,
// at K step ks, its 16 bytes at 32 ks + 16 h: the B operand layout of the
// 32x32x16 MFMA. The ring slot of K step ks is ks % PD; the last steps of a
// tile load the first PD steps of the wave's next tile (or re-read the same
// tile after the last one; those loads are never used). Scores are
// w * ReLU(q . k) (DSA with one head) or w * (q . k), computed as
// fma(w, x, +0) so that a zero product is +0.
template <class C, class Src, class Sink>
__device__ __forceinline__ void wide_scan(const ScoreArgs& a, const Src& src, int kbeg, int kend,
                                          const uint8_t* qlds, const float (&wv)[C::NI], Sink& sink) {
  const int l = lane_id(), h = l >> 5, r32 = l & 31;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
  const int ntiles = kend > kbeg ? (kend - kbeg + C::KT - 1) / C::KT : 0;
  if (wave >= ntiles) return;
  const uint8_t* keys = static_cast<const uint8_t*>(a.keys);
  auto row_of = [&](int tile) {
    const int i = min(kbeg + tile * C::KT + r32, kend - 1);
    return keys + (int64_t)src.key(i) * C::ROWB + h * 16;
  };
  auto ldb = [](const uint8_t* p) { return *reinterpret_cast<const wbf16x8_t*>(p); };
  const uint8_t* rp = row_of(wave);
  wbf16x8_t bq[C::PD];
  wstatic_for<C::PD>([&](auto J) { bq[J] = ldb(rp + J * 32); });
  for (int t = wave; t < ntiles; t += C::WAVES) {
    const int tn = t + C::WAVES < ntiles ? t + C::WAVES : t;
    const uint8_t* np = row_of(tn);
    // the A fragments are the same every tile; an opaque offset keeps the
    // compiler from hoisting all of them (KS * MT * 4 VGPRs) out of the loop
    int qoff = l * 16;
    asm volatile("" : "+v"(qoff));
    const uint8_t* qa = qlds + qoff;
    wf32x16_t acc[C::MT];
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt) acc[mt] = wf32x16_t{};
    wstatic_for<C::KS>([&](auto KSI) {
      constexpr int ks = decltype(KSI)::value;
      const wbf16x8_t b = bq[ks % C::PD];
      wstatic_for<C::MT>([&](auto MTI) {
        constexpr int mt = decltype(MTI)::value;
        const wbf16x8_t af = *reinterpret_cast<const wbf16x8_t*>(qa + (mt * C::KS + ks) * (kWave * 16));
        acc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, b, acc[mt], 0, 0, 0);
      });
      // after every 4th K step, the 4 slots just freed take the loads of
      // steps PD - 3 .. PD ahead: the 4 loads that share each 128-byte line
      // of a row go out back to back, so the line is fetched once instead
      // of being evicted between them (1.25x the HBM rate of one load per
      // step)
      if constexpr (ks % C::LG == C::LG - 1) {
        wstatic_for<C::LG>([&](auto J) {
          constexpr int nx = ks - (C::LG - 1) + J + C::PD;
          if constexpr (nx < C::KS) bq[nx % C::PD] = ldb(rp + nx * 32);
          else bq[nx % C::PD] = ldb(np + (nx - C::KS) * 32);
        });
      }
    });
    // Issue order: the A fragments one K step ahead, then per K step its two
    // MFMAs and the next step's A fragments, with the B loads of the group
    // after every LG-th step. Left alone, the scheduler sinks each B load
    // down to its use, which collapses the ring to one or two fragments in
    // flight.
    __builtin_amdgcn_sched_group_barrier(0x100, C::MT, 0);  // DS read
    wstatic_for<C::KS>([&](auto KSI) {
      __builtin_amdgcn_sched_group_barrier(0x008, C::MT, 0);  // MFMA
      if constexpr (decltype(KSI)::value % C::LG == C::LG - 1)
        __builtin_amdgcn_sched_group_barrier(0x020, C::LG, 0);  // VMEM read
      __builtin_amdgcn_sched_group_barrier(0x100, C::MT, 0);  // DS read
    });
    float sc[C::NI];
#pragma unroll
    for (int it = 0; it < C::NI; ++it) {
      const float x = acc[it >> 4][it & 15];
      sc[it] = fmaf(wv[it], C::RELU ? __builtin_elementwise_maximum(x, 0.0f) : x, 0.0f);
    }
    sink.consume(kbeg + t * C::KT, kend, sc);
    rp = np;
  }
}

// ---------------------------------------------------------------------------
// Sinks. consume(k0, kend, sc) runs after a tile's MFMAs with the lane's
// scores of positions k0 + lane % 32.
// ---------------------------------------------------------------------------

// Every score to out[t * ld + position] (sample and dense scorers).
template <class C>
struct WideDenseSink {
  float* out;
  int64_t ld;
  int qbase, nq;
  __device__ void consume(int k0, int kend, const float (&sc)[C::NI]) {
    const int h = lane_id() >> 5, pos = k0 + (lane_id() & 31);
    if (pos >= kend) return;
#pragma unroll
    for (int it = 0; it < C::NI; ++it) {
      const int t = qbase + wq_of(it, h);
      if (t < nq) out[(int64_t)t * ld + pos] = sc[it];
    }
  }
};

// The scores of one query (the fallback's re-score): item it_t of half h_t.
template <class C>
struct WideRowSink {
  float* out;
  int it_t, h_t;
  __device__ void consume(int k0, int kend, const float (&sc)[C::NI]) {
    const int h = lane_id() >> 5, pos = k0 + (lane_id() & 31);
    float v = 0.0f;
#pragma unroll
    for (int it = 0; it < C::NI; ++it)
      if (it == it_t) v = sc[it];
    if (h == h_t && pos < kend) out[pos] = v;
  }
};

__device__ __forceinline__ int wload(const int* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Fused filter with the row state shared by all key splits (see the top of
// the file). Lane q holds the state of query qbase + q: bin map (delta, c),
// visible range [s, e), current threshold bin tau and its score-domain gate
// T (the GroupedSink bound: bin(fma(I, delta, c)) >= tau holds for every
// I >= (tau - c) / delta, lowered by far more than its rounding error, so a
// compare never drops a key whose bin is >= tau; a key let through just below
// the bin edge is written and counted in its true bin). tq[it] is T of the
// query of item it in the lane's half.
template <class C>
struct WideFusedSink {
  float delta_v, c_v, t_v;
  int tau_v, e_v, s_v;
  float tq[C::NI];
  bool ungated;         // some row of the block has no gate (tau = -1)
  int rq;               // row whose histogram and published bin were read last tile (-1: none)
  int rturn;            // the next of this wave's rows to refresh
  int fturn;            // the next of this wave's rows to flush
  int rg;               // its published bin as read
  int gv;               // the published bin of query qbase + lane, read with it
  int rcount;           // tiles consumed
  uint32_t rh[4];       // its shared histogram, bins 4 * lane .. + 3
  int* gate;            // [nq] published threshold bins
  uint32_t* hist;       // [nq, m] shared histograms
  lds_u32_t* bh;        // [64, m] LDS: block counts not yet moved to `hist`
  lds_i32_t* btau;      // [64] LDS: the block's threshold bins
  lds_u32_t* btail;     // [64] LDS: slots taken in the block's list of each row
  float2* bmap;         // [64] LDS: bin map (delta, c) of each row
  int vis_s, vis_e;     // every row of the block sees [vis_s, vis_e)
  int2* cand;           // [nq, S, cap] (key, score) lists, this block's is `split`
  int qbase, nq, S, split, cap, m, k;

  __device__ static float gate_floor(float delta, float c, int tau) {
    if (tau < 0) return -__builtin_inff();
    const float t = (float)tau, i0 = (t - c) / delta;
    const float err = ((fabsf(t) + fabsf(c)) / delta + fabsf(i0)) * 0x1p-20f;
    return i0 - err;
  }

  __device__ void init(const ScoreArgs& a, const RowParam* params, int kend) {
    const int l = lane_id(), t = qbase + l;
    RowRange rr{0, 0};
    float dl = 1.0f, c = 0.0f;
    int t0 = -1;
    if (t < nq) {
      rr = row_range(a.offs, a.starts, t, a.nk);
      const RowParam p = params[t];
      dl = p.delta;
      c = p.c;
      t0 = p.tau0;
    }
    e_v = rr.e < kend ? rr.e : kend;
    s_v = rr.s;
    delta_v = dl;
    c_v = c;
    tau_v = t0;
    // each wave writes the whole map (the same values) before its own reads
    bmap[l] = make_float2(dl, c);
    int cs = t < nq ? rr.s : 0, ce = t < nq ? e_v : INT_MAX;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      cs = max(cs, __shfl_xor(cs, o));
      ce = min(ce, __shfl_xor(ce, o));
    }
    vis_s = __builtin_amdgcn_readfirstlane(cs);
    vis_e = __builtin_amdgcn_readfirstlane(ce);
    rq = -1;
    rcount = (int)(threadIdx.x / kWave) % C::REFRESH;
    // wave w refreshes rows w, w + WAVES, ...; blocks start at different ones
    rturn = (int)(threadIdx.x / kWave) + C::WAVES * (int)(blockIdx.x % (C::QT / C::WAVES));
    fturn = (rturn + C::WAVES * (C::QT / C::WAVES / 2)) & (C::QT - 1);
    update_gates();
  }

  __device__ void update_gates() {
    const int l = lane_id(), h = l >> 5;
    const bool valid = qbase + l < nq;
    t_v = valid ? gate_floor(delta_v, c_v, tau_v) : __builtin_inff();
    ungated = __ballot(valid && tau_v < 0) != 0;
    wstatic_for<C::NI>([&](auto I) {
      constexpr int it = decltype(I)::value;
      const float x0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, t_v), wq_of(it, 0)));
      const float x1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, t_v), wq_of(it, 1)));
      tq[it] = h ? x1 : x0;
    });
  }


  // the threshold bin of row qbase + rq from its histogram read one tile
  // ago: into the block's bins, and published when it beats the published one
  __device__ void finish_refresh() {
    const int b = wave_threshold_vals(rh, (uint32_t)k, nullptr);
    const int l = lane_id();
    // every row's published bin, and this row's own result, into the block's
    const int nb = l == rq ? max(b, gv) : gv;
    if (nb > btau[l]) __hip_atomic_fetch_max(btau + l, nb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    if (l == 0 && b > rg) __hip_atomic_fetch_max(gate + qbase + rq, b, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    rq = -1;
  }

  // move the block's counts of row qbase + q to the shared histogram (each
  // LDS bin swapped with 0, so counts other waves add meanwhile stay for the
  // next move), then read the shared histogram and the published bin
  // Counts in bins below the block's current bin of the row are dropped:
  // that bin never exceeds the final threshold bin, and only bins at or
  // above the final one are ever read (the refresh walks stop there too).
  __device__ void flush(int q) {
    uint32_t* hr = hist + (int64_t)(qbase + q) * m;
    const int l = lane_id(), bt = btau[q];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int b = 4 * l + j;
      if (b < m && b >= bt) {
        const uint32_t v = __hip_atomic_exchange(bh + q * m + b, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        if (v) __hip_atomic_fetch_add(hr + b, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }

  __device__ void start_refresh(int q) {
    uint32_t* hr = hist + (int64_t)(qbase + q) * m;
    const int l = lane_id();
    flush(q);
    // one device-coherent 16-byte read per lane (bins past m read as 0: the
    // buffer covers the row only)
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(hr, 0, m * 4, kBufferRaw);
    const wu32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(rs, l * 16, 0, kCoherent);
#pragma unroll
    for (int j = 0; j < 4; ++j) rh[j] = 4 * l + j < m ? v[j] : 0u;
    gv = qbase + l < nq ? wload(gate + qbase + l) : -1;
    rg = __builtin_amdgcn_readlane(gv, q);
    rq = q;
  }

  __device__ bool lane_pass(int it, int key, uint32_t bits, int qa, int qb) const {
    const int h = lane_id() >> 5;
    const int ea = __builtin_amdgcn_readlane(e_v, qa), eb = __builtin_amdgcn_readlane(e_v, qb);
    const int sa = __builtin_amdgcn_readlane(s_v, qa), sb = __builtin_amdgcn_readlane(s_v, qb);
    return ((bits >> it) & 1u) && key < (h ? eb : ea) && key >= (h ? sb : sa);
  }

  // write-back of the items in `items` (wave-uniform bit set of score items
  // some lane passed; bits = this lane's): every passing lane takes its slot
  // in the block's list of its row with an LDS atomic and reads the row's bin
  // map from LDS; the visible range is checked only on tiles that cross some
  // row's range
  __device__ void emit(int key, uint32_t bits, uint32_t items, const float (&sc)[C::NI]) {
    typedef float fNI __attribute__((ext_vector_type(C::NI)));
    const int l = lane_id(), h = l >> 5;
    const int k0 = key - (l & 31);
    const bool inside = k0 >= vis_s && k0 + C::KT <= vis_e;
    fNI scv;
#pragma unroll
    for (int it = 0; it < C::NI; ++it) scv[it] = sc[it];
    for (uint32_t rem = items; rem; rem &= rem - 1) {
      const int it = __builtin_ctz(rem), qa = wq_of(it, 0), qb = qa + 4;
      const bool pass = inside ? ((bits >> it) & 1u) != 0u : lane_pass(it, key, bits, qa, qb);
      if (pass) {
        const int q = h ? qb : qa;
        const uint32_t pos = __hip_atomic_fetch_add(btail + q, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        const float2 mp = bmap[q];
        const float s = scv[it];
        const int64_t t = qbase + q;
        if (pos < (uint32_t)cap) cand[ilv_index(t * S + split, pos, (int64_t)nq * S)] = make_int2(key, __float_as_int(s));
        // counted only when x >= 0 (not NaN, not below the range): the add is
        // issued either way, of 0 for the others
        const float x = fmaf(s, mp.x, mp.y);
        const int b = min(max(__float2int_rz(x), 0), m - 1);
        __hip_atomic_fetch_add(bh + q * m + b, x >= 0.0f ? 1u : 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      }
    }
  }

  __device__ void consume(int k0, int kend, const float (&sc)[C::NI]) {
    const int l = lane_id(), key = k0 + (l & 31);
    // 1. thresholds: finish this wave's refresh begun one tile ago, then take
    //    the block's bins
    if (rq >= 0) finish_refresh();
    const int bt = btau[l];
    if (__ballot(bt > tau_v) != 0) {
      tau_v = max(tau_v, bt);
      update_gates();
    }
    // 2. gate. Fast path on the vector ALU: the largest margin score - T of
    //    the lane (a NaN score only matters to an ungated row, and then the
    //    fast path is skipped)
    bool any = true;
    if (!ungated) {
      float mx = -__builtin_inff();
#pragma unroll
      for (int it = 0; it < C::NI; ++it) mx = fmaxf(mx, sc[it] - tq[it]);
      any = __ballot(mx >= 0.0f) != 0;
    }
    if (any) {
      uint32_t bits = 0;
#pragma unroll
      for (int it = 0; it < C::NI; ++it) bits |= !(sc[it] < tq[it]) ? (1u << it) : 0u;
      if (key >= kend) bits = 0;
      const uint32_t items = wave_or(bits);
      if (items) emit(key, bits, items, sc);
    }
    // 3. move the counts of one of this wave's rows to the shared histogram
    //    every tile; every C::REFRESH tiles (the block's waves in turn)
    //    begin the refresh of another
    const int qf = fturn;
    fturn = (fturn + C::WAVES) & (C::QT - 1);
    if (qbase + qf < nq) flush(qf);
    if (++rcount % C::REFRESH != 0) return;
    const int q = rturn;
    rturn = (rturn + C::WAVES) & (C::QT - 1);
    if (qbase + q < nq) start_refresh(q);
  }
};

// ---------------------------------------------------------------------------
// Kernels
// ---------------------------------------------------------------------------
template <class C>
__global__ __launch_bounds__(C::NTHREADS) void k_wide_sample(ScoreArgs a, const int32_t* list, int ns, float* samp,
                                                             int slice) {
  extern __shared__ __align__(16) uint8_t lds[];
  const int q0 = blockIdx.x * C::QT;
  const int kb = blockIdx.y * slice, ke = min(kb + slice, ns);
  wide_load_q<C>(lds, a, q0);
  float wv[C::NI];
  wide_weights<C>(wv, a, q0);
  WideDenseSink<C> sink{samp, ns, q0, a.nq};
  wide_scan<C>(a, WSrcList{list}, kb, ke, lds, wv, sink);
}

template <class C>
__global__ __launch_bounds__(C::NTHREADS) void k_wide_dense(ScoreArgs a, float* out, int64_t ld, int slice) {
  extern __shared__ __align__(16) uint8_t lds[];
  const int q0 = blockIdx.x * C::QT;
  const int kb = blockIdx.y * slice, ke = min(kb + slice, a.nk);
  wide_load_q<C>(lds, a, q0);
  float wv[C::NI];
  wide_weights<C>(wv, a, q0);
  WideDenseSink<C> sink{out, ld, q0, a.nq};
  wide_scan<C>(a, WSrcContig{}, kb, ke, lds, wv, sink);
}

// Shared row state: empty histograms, published bins = the sample's.
__global__ void k_wide_init(const RowParam* params, int nq, int m, int* gate, uint32_t* hist) {
  const int64_t n = (int64_t)nq * m, stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (int64_t i = i0; i < n; i += stride) hist[i] = 0u;
  for (int64_t i = i0; i < nq; i += stride) gate[i] = params[i].tau0;
}

template <class C>
__global__ __launch_bounds__(C::NTHREADS) void k_wide_fused(ScoreArgs a, const RowParam* params, int S, int L, int cap,
                                                            int m, int k, int* gate, uint32_t* cnt, uint32_t* hist,
                                                            int2* cand) {
  extern __shared__ __align__(16) uint8_t lds[];
  int* rng = reinterpret_cast<int*>(lds + C::Q_LDS);  // [0] largest end, [1] smallest start
  uint32_t* btail = reinterpret_cast<uint32_t*>(lds + C::Q_LDS + 16);            // [QT]
  int* btau = reinterpret_cast<int*>(lds + C::Q_LDS + 16 + C::QT * 4);           // [QT]
  float2* bmap = reinterpret_cast<float2*>(lds + C::Q_LDS + 16 + C::QT * 8);     // [QT]
  uint32_t* bh = reinterpret_cast<uint32_t*>(lds + C::Q_LDS + 16 + C::QT * 16);  // [QT, m]
  const int tile = blockIdx.x / S, split = blockIdx.x - tile * S, q0 = tile * C::QT;
  if (threadIdx.x == 0) {
    rng[0] = 0;
    rng[1] = a.nk;
  }
  if (threadIdx.x < C::QT) {
    btail[threadIdx.x] = 0u;
    btau[threadIdx.x] = q0 + (int)threadIdx.x < a.nq ? params[q0 + threadIdx.x].tau0 : -1;
  }
  for (int i = threadIdx.x; i < C::QT * m; i += C::NTHREADS) bh[i] = 0u;
  __syncthreads();
  if (threadIdx.x < C::QT && q0 + (int)threadIdx.x < a.nq) {
    const RowRange rr = row_range(a.offs, a.starts, q0 + threadIdx.x, a.nk);
    if (rr.e > rr.s) {
      atomicMax(&rng[0], rr.e);
      atomicMin(&rng[1], rr.s);
    }
  }
  wide_load_q<C>(lds, a, q0);  // ends with a barrier
  // the split's keys within the union of the block's rows' ranges
  const int kb = max(split * L, rng[1]);
  const int ke = min(min(split * L + L, a.nk), rng[0]);
  float wv[C::NI];
  wide_weights<C>(wv, a, q0);
  WideFusedSink<C> sink;
  sink.gate = gate;
  sink.hist = hist;
  sink.bh = (lds_u32_t*)bh;
  sink.btau = (lds_i32_t*)btau;
  sink.btail = (lds_u32_t*)btail;
  sink.bmap = bmap;
  sink.cand = cand;
  sink.qbase = q0;
  sink.nq = a.nq;
  sink.S = S;
  sink.split = split;
  sink.cap = cap;
  sink.m = m;
  sink.k = k;
  sink.init(a, params, ke);
  wide_scan<C>(a, WSrcContig{}, kb, ke, lds, wv, sink);
  __syncthreads();
  if (threadIdx.x < C::QT && q0 + (int)threadIdx.x < a.nq)
    cnt[(int64_t)(q0 + threadIdx.x) * S + split] = btail[threadIdx.x];
  // the counts no flush has moved yet (bins at or above the block's bin)
  for (int i = threadIdx.x; i < C::QT * m; i += C::NTHREADS) {
    const int q = i / m;
    if (bh[i] != 0u && q0 + q < a.nq && i - q * m >= btau[q])
      __hip_atomic_fetch_add(hist + (int64_t)(q0 + q) * m + (i - q * m), bh[i], __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Exact fallback for queued rows: the row's visible range re-scored into a
// scratch row, then radix-selected. Split mode (few rows, fallback_chunks > 1):
// one block per (queue entry, chunk of the row's keys) writing into the
// entry's scratch row and selecting the chunk's top-k into the candidate
// arrays (cidx, cscore); the block that counts the row's last chunk selects
// the row from them. Otherwise the first `slots` blocks take one whole row at
// a time, each into its own scratch row. One loop serves both (one item per
// block in split mode).
template <class C>
__global__ __launch_bounds__(C::NTHREADS) void k_wide_fallback(ScoreArgs a, int k, uint32_t flags, uint32_t* qctl,
                                                               const int32_t* queue, int slots, float* scratch,
                                                               int32_t* cidx, float* cscore, int32_t* out_i,
                                                               float* out_s) {
  extern __shared__ __align__(16) uint8_t lds[];
  __shared__ int last;
  const uint32_t n = qctl[0];
  const int chunks = fallback_chunks(n, gridDim.x, slots, a.nk);
  const int active = chunks > 1 ? (int)gridDim.x : min((int)gridDim.x, slots);
  const uint32_t items = n * (uint32_t)chunks;
  if ((int)blockIdx.x >= active) return;
  for (uint32_t it = blockIdx.x; it < items; it += (uint32_t)active) {
    const int e = (int)(it / (uint32_t)chunks), c = (int)it - e * chunks;
    const int row = queue[e];
    const RowRange rr = row_range(a.offs, a.starts, row, a.nk);
    const int len = rr.e > rr.s ? rr.e - rr.s : 0;
    const int per = ((len + chunks - 1) / chunks + C::STEP - 1) / C::STEP * C::STEP;
    const int kb = min(rr.s + c * per, rr.s + len), ke = min(kb + per, rr.s + len);
    float* srow = scratch + (int64_t)(chunks > 1 ? e : (int)blockIdx.x) * a.nk;
    const int q0 = (row / C::QT) * C::QT, ql = row - q0;
    wide_load_q<C>(lds, a, q0);
    float wv[C::NI];
    wide_weights<C>(wv, a, q0);
    WideRowSink<C> sink{srow, 16 * (ql >> 5) + 4 * ((ql & 31) >> 3) + (ql & 3), (ql >> 2) & 1};
    wide_scan<C>(a, WSrcContig{}, kb, ke, lds, wv, sink);
    __threadfence_block();
    __syncthreads();
    if (chunks > 1) {
      const int64_t cb = (int64_t)e * chunks * k;
      split_fallback_select<C::NTHREADS>(srow, rr.s, len, per, chunks, c, kb, ke, k, cidx + cb, cscore + cb,
                                         &qctl[kQctlDone + e], out_i + (int64_t)row * k, out_s + (int64_t)row * k,
                                         flags & LT_SORTED_OUTPUT, lds, &last);
    } else {
      radix_select_row<C::NTHREADS>(srow + rr.s, len, k, out_i + (int64_t)row * k, out_s + (int64_t)row * k,
                                    flags & LT_SORTED_OUTPUT, lds, rr.s);
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Variants and launchers
// ---------------------------------------------------------------------------
//                  d   ReLU
#define LT_WIDE_VARIANTS(X) \
  X(768, false)             \
  X(768, true)

template <class F>
static bool with_wide(int dt, int mode, int h, int d, F&& f) {
  if (dt != LT_BF16 || h != 1) return false;
  const bool relu = mode == LT_SCORE_DSA;
#define LT_WCASE(D, RELU)                          \
  if (d == D && relu == RELU) {                    \
    f.template operator()<WCfg<D, RELU>>();        \
    return true;                                   \
  }
  LT_WIDE_VARIANTS(LT_WCASE)
#undef LT_WCASE
  return false;
}

template <class K>
static void allow_lds(K kernel, size_t bytes) {
  if (bytes > 65536) (void)hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

ScoreShape wide_shape(int dtype, int mode, int h, int d) {
  ScoreShape s{0, 0, 0, 0, 0, 0, 0};
  with_wide(dtype, mode, h, d, [&]<class C>() {
    s.supported = 1;
    s.queries_per_block = C::QT;
    s.keys_per_step = C::STEP;
    s.threads = C::NTHREADS;
    s.scan_lds = C::Q_LDS + 16 + C::QT * 16;  // queries, key range, list tails, bins, bin maps
    s.shared_rows = 1;
    s.arrival_order = 1;
  });
  return s;
}

static constexpr int kWideSlice = 8192;      // positions per block in the dense scorer
static constexpr int kWideSampleBlocks = 256;

hipError_t launch_wide_sample(const ScoreArgs& a, const int32_t* list, int ns, float* samp, hipStream_t st) {
  hipError_t err = hipErrorInvalidValue;
  with_wide(a.dtype, a.mode, a.h, a.d, [&]<class C>() {
    const int tiles = (a.nq + C::QT - 1) / C::QT;
    const int want = tiles > 0 ? (kWideSampleBlocks + tiles - 1) / tiles : 1;
    int slice = (ns + want - 1) / want;
    slice = ((slice + C::STEP - 1) / C::STEP) * C::STEP;
    slice = slice < C::STEP ? C::STEP : (slice > kWideSlice ? kWideSlice : slice);
    const dim3 grid(tiles, (ns + slice - 1) / slice);
    if (grid.x == 0 || grid.y == 0) {
      err = hipSuccess;
      return;
    }
    allow_lds(k_wide_sample<C>, C::Q_LDS);
    hipLaunchKernelGGL(k_wide_sample<C>, grid, dim3(C::NTHREADS), C::Q_LDS, st, a, list, ns, samp, slice);
    err = hipGetLastError();
  });
  return err;
}

hipError_t launch_wide_dense(const ScoreArgs& a, float* out, int64_t ld, hipStream_t st) {
  hipError_t err = hipErrorInvalidValue;
  with_wide(a.dtype, a.mode, a.h, a.d, [&]<class C>() {
    const dim3 grid((a.nq + C::QT - 1) / C::QT, (a.nk + kWideSlice - 1) / kWideSlice);
    if (grid.x == 0 || grid.y == 0) {
      err = hipSuccess;
      return;
    }
    allow_lds(k_wide_dense<C>, C::Q_LDS);
    hipLaunchKernelGGL(k_wide_dense<C>, grid, dim3(C::NTHREADS), C::Q_LDS, st, a, out, ld, kWideSlice);
    err = hipGetLastError();
  });
  return err;
}

hipError_t launch_wide_fused(const ScoreArgs& a, const RowParam* params, int S, int L, int cap, int m, int k,
                             int* gate, uint32_t* cnt, uint32_t* hist, int2* cand, hipStream_t st) {
  hipError_t err = hipErrorInvalidValue;
  with_wide(a.dtype, a.mode, a.h, a.d, [&]<class C>() {
    const int tiles = (a.nq + C::QT - 1) / C::QT;
    if (tiles == 0) {
      err = hipSuccess;
      return;
    }
    const int64_t n = (int64_t)a.nq * m;
    const int ib = (int)std::min<int64_t>((n + 255) / 256, 1024);
    hipLaunchKernelGGL(k_wide_init, dim3(ib < 1 ? 1 : ib), dim3(256), 0, st, params, a.nq, m, gate, hist);
    if ((err = hipGetLastError()) != hipSuccess) return;
    const size_t lds = C::Q_LDS + 16 + C::QT * 16 + (size_t)C::QT * m * 4;
    allow_lds(k_wide_fused<C>, lds);
    hipLaunchKernelGGL(k_wide_fused<C>, dim3(tiles * S), dim3(C::NTHREADS), lds, st, a, params, S, L, cap, m, k,
                       gate, cnt, hist, cand);
    err = hipGetLastError();
  });
  return err;
}

hipError_t launch_wide_fallback(const ScoreArgs& a, int k, uint32_t flags, uint32_t* qctl, const int32_t* queue,
                                int slots, float* scratch, int32_t* cidx, float* cscore, int32_t* out_i, float* out_s,
                                hipStream_t st) {
  hipError_t err = hipErrorInvalidValue;
  with_wide(a.dtype, a.mode, a.h, a.d, [&]<class C>() {
    size_t lds = C::Q_LDS;
    const size_t rl = radix_lds_bytes(k);
    if (rl > lds) lds = rl;
    allow_lds(k_wide_fallback<C>, lds);
    hipLaunchKernelGGL(k_wide_fallback<C>, dim3(kFallbackGrid), dim3(C::NTHREADS), lds, st, a, k, flags, qctl,
                       queue, slots, scratch, cidx, cscore, out_i, out_s);
    err = hipGetLastError();
  });
  return err;
}

}  // namespace lt
