// Score-side kernels (gfx950): the index score of Eq. (1) on MFMA matrix
// cores with the ReLU / head-weighted epilogue in registers, driven by one
// LDS-tiled key scan that feeds four consumers:
//   * the sample scorer (sec. 3.2 "Sampling"),
//   * the dense scorer (the materialising baseline, sec. 1),
//   * the fused filter scan (sec. 3.2 "Filtering" + "Threshold Refresh"),
//   * the exact fallback for overflowed rows.
// All four share the same arithmetic, so their scores are bit-identical.
//
// Layout of the contraction. A block owns QT = WAVES * QW queries and streams
// the keys through LDS in tiles of KT = 32 * NT keys (double-buffered). Each
// wave owns QW queries and keeps their QW * H head vectors stationary in VGPRs
// as the A operand (rows = (query, head), 32 per M tile); the key tile is the B
// operand (columns = keys). With 32x32 MFMA tiles each lane ends up holding 16
// heads of one key column per M tile, so the head reduction of Eq. (1) is an
// in-lane chain of ReLU + FMA, plus (for H >= 8) one exchange between the two
// 32-lane halves, arranged so that after it every lane holds a full score.
#include <utility>

#include <type_traits>

#include "internal.hpp"
#include "select_dev.hpp"

namespace lt {

enum { DT_F32 = LT_F32, DT_BF16 = LT_BF16, DT_FP8 = LT_FP8_E4M3FN };

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef int i32x8_t __attribute__((ext_vector_type(8)));
typedef int i32x4_t __attribute__((ext_vector_type(4)));

template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  [&]<int... I>(std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
  }(std::make_integer_sequence<int, N>{});
}

// ---------------------------------------------------------------------------
// MFMA flavours. Each lane feeds FB bytes = KI/2 consecutive elements of its
// row (A) or column (B) per instruction: elements [KI/2 * (lane / 32), +KI/2)
// of the K slice. A and B use the same lane->k assignment, so the instruction
// sums every product of the slice exactly once.
// ---------------------------------------------------------------------------
template <int DT>
struct Mfma;

template <>
struct Mfma<DT_F32> {
  static constexpr int KI = 2, ES = 4, FB = 4;
  using Frag = float;
  __device__ static Frag load(const uint8_t* p) { return *reinterpret_cast<const float*>(p); }
  __device__ static Frag zero() { return 0.0f; }
  __device__ static f32x16_t mma(Frag a, Frag b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

template <>
struct Mfma<DT_BF16> {
  static constexpr int KI = 16, ES = 2, FB = 16;
  using Frag = bf16x8_t;
  __device__ static Frag load(const uint8_t* p) { return *reinterpret_cast<const bf16x8_t*>(p); }
  __device__ static Frag zero() { return __builtin_bit_cast(bf16x8_t, i32x4_t{0, 0, 0, 0}); }
  __device__ static f32x16_t mma(Frag a, Frag b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};

template <>
struct Mfma<DT_FP8> {
  static constexpr int KI = 64, ES = 1, FB = 32;
  using Frag = i32x8_t;
  __device__ static Frag load2(const uint8_t* p0, const uint8_t* p1) {
    i32x4_t lo = *reinterpret_cast<const i32x4_t*>(p0);
    i32x4_t hi = *reinterpret_cast<const i32x4_t*>(p1);
    return i32x8_t{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  }
  __device__ static Frag load(const uint8_t* p) { return load2(p, p + 16); }
  __device__ static Frag zero() { return i32x8_t{0, 0, 0, 0, 0, 0, 0, 0}; }
  // OCP E4M3 for both operands (format code 0), unit block scales (E8M0 127).
  __device__ static f32x16_t mma(Frag a, Frag b, f32x16_t c) {
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 127, 0, 127);
  }
};

// ---------------------------------------------------------------------------
// Static configuration of one (dtype, H, d) variant.
// ---------------------------------------------------------------------------
template <int DT_, int H_, int D_, int QW_, int NT_, int WAVES_, bool RELU_, bool UNITW_ = false>
struct Cfg {
  using M = Mfma<DT_>;
  static constexpr int DT = DT_, H = H_, D = D_, QW = QW_, NT = NT_, WAVES = WAVES_;
  static constexpr bool RELU = RELU_;
  // one head, no ReLU and no head weights (w = NULL): the score is the dot
  // product itself, taken from the accumulator with no epilogue arithmetic
  // (the weighted form fmaf(1, x, +0) gives the same bits: an accumulator
  // that starts at +0 never holds -0)
  static constexpr bool UNITW = UNITW_;
  static_assert(!UNITW || (H == 1 && !RELU), "unit weights: one head, inner product");
  static constexpr int MT = QW * H / 32;               // M tiles per wave
  static constexpr int KS = D / M::KI;                 // K steps per key
  static constexpr int KT = 32 * NT;                   // keys per tile
  static constexpr int QT = WAVES * QW;                // queries per block
  static constexpr int ROWB = D * M::ES;               // bytes per key row
  static constexpr int TILE_BYTES = KT * ROWB;         // LDS tile: rows of 16-B chunks, XOR-swizzled
  static constexpr int RING = 4;                       // LDS tiles in flight
  // fp8: the key scales of each tile follow the tiles into LDS, in a ring of
  // twice as many slots (the epilogue of tile t runs one step after its MFMAs,
  // when the tile's own slot is already being refilled)
  static constexpr int SCALE_RING = 2 * RING;
  static constexpr int SCALE_BYTES = DT == DT_FP8 ? SCALE_RING * KT * 4 : 0;
  static constexpr int SCAN_LDS = RING * TILE_BYTES + SCALE_BYTES;
  static constexpr int CPK = ROWB / 16;                // 16-byte chunks per key
  // XOR swizzle key of row n: the 16 lanes of one LDS access group read the
  // same chunk of 16 consecutive rows and must hit 16 distinct 16-byte bank
  // slots of a 256-byte bank line; rows shorter than 256 bytes share a line,
  // so consecutive rows that do are told apart by the line they sit in
  static constexpr int RPL = ROWB >= 256 ? 1 : 256 / ROWB;  // rows per bank line
  __host__ __device__ static constexpr int swz(int n) { return n / RPL; }
  static constexpr int CHUNKS = KT * CPK;
  static constexpr int NTHREADS = WAVES * kWave;
  static constexpr int CPT = CHUNKS / NTHREADS;      // staged chunks per thread per tile
  // GROUPED: H <= 4, a 4-row accumulator group holds whole queries, no
  // cross-lane step. Otherwise H % 8 == 0 and the halves are combined.
  static constexpr bool GROUPED = H <= 4;
  static constexpr int GPQ = GROUPED ? 4 / H : 1;      // queries per 4-row group
  static constexpr int NI = GROUPED ? NT * MT * 4 * GPQ : NT * QW / 2;  // scores per lane per tile
  static constexpr int NIH = GROUPED ? MT * 4 * GPQ : QW;              // per-lane results of one sub-tile
  // epilogue VALU ops of one sub-tile (ReLU + FMA per accumulator element)
  // spread over the MFMAs of the other sub-tile. The 64-head values leave
  // room for the combine and gate work of the half step too (measured best
  // on MI355X: 5 for bf16, against 4 for the epilogue alone).
#ifndef LT_FP8_VALU_PER_MFMA
#define LT_FP8_VALU_PER_MFMA 20
#endif
#ifndef LT_BF16_VALU_PER_MFMA
#define LT_BF16_VALU_PER_MFMA 5
#endif
  static constexpr int VALU_PER_MFMA = H == 64 && QW == 1 && DT == DT_BF16  ? LT_BF16_VALU_PER_MFMA
                                       : H == 64 && QW == 1 && DT == DT_FP8 ? LT_FP8_VALU_PER_MFMA
                                                                            : (32 * MT + KS * MT - 1) / (KS * MT);
  static_assert((QW * H) % 32 == 0, "a wave must fill whole M tiles");
  static_assert(NT == 2, "the scan pipelines the two 32-key halves of a tile");
  static_assert(CHUNKS % NTHREADS == 0 && CPT < 16, "tile staging assumes whole instructions per thread");
  static_assert((CPK & (CPK - 1)) == 0, "chunks per key row must be a power of two");
  static_assert(D % M::KI == 0, "head dim must be a multiple of the MFMA K");
  static_assert(ROWB % 16 == 0, "key rows must be a multiple of 16 bytes");
  static_assert(GROUPED ? (4 % H == 0) : (H % 8 == 0 && (NT * QW) % 2 == 0), "unsupported head layout");

  // Score item `it` of a lane in half h (0: lanes 0-31, 1: lanes 32-63):
  // which of the wave's queries and which 32-key sub-tile it belongs to.
  __host__ __device__ static constexpr int item_q(int it, int h) {
    if constexpr (GROUPED) {
      const int s = it % GPQ, g = it / GPQ, i = g % 4, mt = (g / 4) % MT;
      return (32 * mt + 8 * i + 4 * h + s * H) / H;
    } else {
      return (2 * it + h) / NT;
    }
  }
  __host__ __device__ static constexpr int item_nt(int it, int h) {
    if constexpr (GROUPED) return it / (MT * 4 * GPQ);
    else return (2 * it + h) % NT;
  }
};

// Per-wave stationary operands: the A fragments of the wave's queries and the
// head weight of every accumulator row the lane holds.

template <class C>
struct WaveQ {
  typename C::M::Frag qa[C::MT][C::KS];
  float wv[C::MT][16];
};

template <class C>
__device__ __forceinline__ void load_q(WaveQ<C>& s, const ScoreArgs& a, int qbase) {
  using M = typename C::M;
  const int l = lane_id(), h = l >> 5, r32 = l & 31;
  const uint8_t* q = static_cast<const uint8_t*>(a.q);
#pragma unroll
  for (int mt = 0; mt < C::MT; ++mt) {
    const int r = 32 * mt + r32, ql = r / C::H, j = r % C::H, t = qbase + ql;
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
      if (t < a.nq) {
        const int64_t el = ((int64_t)t * C::H + j) * C::D + ks * M::KI + h * (M::KI / 2);
        s.qa[mt][ks] = M::load(q + el * M::ES);
      } else {
        s.qa[mt][ks] = M::zero();
      }
    }
  }
#pragma unroll
  for (int mt = 0; mt < C::MT; ++mt) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int r = 32 * mt + 8 * (v >> 2) + 4 * h + (v & 3), ql = r / C::H, j = r % C::H, t = qbase + ql;
      float wt = 0.0f;
      if (t < a.nq) {
        wt = a.w ? a.w[(int64_t)t * C::H + j] : 1.0f;
        if constexpr (C::DT == DT_FP8) wt *= a.q_scale[(int64_t)t * C::H + j];
      }
      s.wv[mt][v] = wt;
    }
  }
}

// One half step: q . k for every row of the wave against one 32-key sub-tile.
// acc[mt] is the 32x32 block of M tile mt; accumulator register v of a lane
// is row 8*(v/4) + 4*(lane/32) + v%4 of the M tile, column lane%32.
// LDS tile layout: key row n occupies ROWB contiguous bytes; its 16-byte
// chunk c is stored at chunk slot c ^ (swz(n) mod CPK). The swizzle spreads
// the lanes that read the same chunk of consecutive keys over distinct banks
// without padding, so tiles can be filled by direct HBM -> LDS loads.
template <class C>
__device__ __forceinline__ int lds_offset(int n, int byte) {
  return n * C::ROWB + ((((byte >> 4) ^ C::swz(n)) & (C::CPK - 1)) << 4) + (byte & 15);
}

template <class C>
__device__ __forceinline__ void load_b(const uint8_t* tile, int nt, typename C::M::Frag (&b)[C::KS]) {
  using M = typename C::M;
  const int l = lane_id(), h = l >> 5, r32 = l & 31;
  const int n = nt * 32 + r32;
#pragma unroll
  for (int ks = 0; ks < C::KS; ++ks) {
    const int byte = ks * M::KI * M::ES + h * M::FB;
    if constexpr (M::FB <= 16) {
      b[ks] = M::load(tile + lds_offset<C>(n, byte));
    } else {
      b[ks] = M::load2(tile + lds_offset<C>(n, byte), tile + lds_offset<C>(n, byte + 16));
    }
  }
}

// The same B fragments with the per-lane part of every address held in a
// register (one per 16-byte piece) and the tile slot and sub-tile folded into
// the LDS instruction's immediate offset: row nt * 32 + r sits nt * 32 rows
// after row r with the same swizzle, since 32 / RPL is a multiple of CPK.
template <class C>
struct BLane {
  using M = typename C::M;
  static constexpr int PIECES = M::FB == 32 ? 2 * C::KS : C::KS;
  static constexpr bool ENABLED = (M::FB == 16 || M::FB == 32) && PIECES <= 8;
  uint32_t o[ENABLED ? PIECES : 1];
  // o[j]: LDS address of piece j of this lane in slot 0, sub-tile 0
  __device__ void init(const uint8_t* tiles) {
    if constexpr (ENABLED) {
      static_assert((32 / C::RPL) % C::CPK == 0, "sub-tile offset must keep the swizzle");
      const int l = lane_id(), h = l >> 5, r32 = l & 31;
      const uint32_t base = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint8_t*)tiles;
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) {
        const int byte = ks * M::KI * M::ES + h * M::FB;
        if constexpr (M::FB == 16) {
          o[ks] = base + (uint32_t)lds_offset<C>(r32, byte);
        } else {
          o[2 * ks] = base + (uint32_t)lds_offset<C>(r32, byte);
          o[2 * ks + 1] = base + (uint32_t)lds_offset<C>(r32, byte + 16);
        }
      }
    }
  }
  // new values each tile as far as the compiler knows, so that it folds the
  // slot offsets into the instructions instead of keeping one register per
  // (slot, piece)
  __device__ void opaque() {
    if constexpr (ENABLED) {
#pragma unroll
      for (int j = 0; j < PIECES; ++j) asm volatile("" : "+v"(o[j]));
    }
  }
};

template <class C, int SLOT, int NT>
__device__ __forceinline__ void load_b_at(const uint8_t* tiles, const BLane<C>& bl,
                                          typename C::M::Frag (&b)[C::KS]) {
  using M = typename C::M;
  typedef __attribute__((address_space(3))) const i32x4_t* lds_v4;
  constexpr uint32_t off = SLOT * C::TILE_BYTES + NT * 32 * C::ROWB;
  if constexpr (BLane<C>::ENABLED) {
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
      if constexpr (M::FB == 16) {
        b[ks] = __builtin_bit_cast(typename M::Frag, *(lds_v4)(uintptr_t)(bl.o[ks] + off));
      } else {
        const i32x4_t lo = *(lds_v4)(uintptr_t)(bl.o[2 * ks] + off);
        const i32x4_t hi = *(lds_v4)(uintptr_t)(bl.o[2 * ks + 1] + off);
        b[ks] = typename M::Frag{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      }
    }
  } else {
    load_b<C>(tiles + SLOT * C::TILE_BYTES, NT, b);
  }
}

template <class C>
__device__ __forceinline__ void mma_half(const WaveQ<C>& s, const typename C::M::Frag (&b)[C::KS],
                                         f32x16_t (&acc)[C::MT]) {
  using M = typename C::M;
#pragma unroll
  for (int mt = 0; mt < C::MT; ++mt) acc[mt] = f32x16_t{};
#pragma unroll
  for (int ks = 0; ks < C::KS; ++ks)
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt) acc[mt] = M::mma(s.qa[mt][ks], b[ks], acc[mt]);
}

// ReLU of Eq. (1) as IEEE-754-2019 maximum (one v_maximum3_f32; NaN
// propagates); inner-product mode skips it.
template <class C>
__device__ __forceinline__ float relu(float x) {
  if constexpr (C::RELU) return __builtin_elementwise_maximum(x, 0.0f);
  else return x;
}

// Eq. (1) epilogue of one sub-tile in registers: ReLU of every head's dot
// product and the weighted sum over the heads this lane holds.
//   GROUPED: out[j], j = (mt*4 + i)*GPQ + sq, are complete scores.
//   else:    out[q] is the lane's partial sum for query q (half of the heads).
template <class C>
__device__ __forceinline__ void reduce_half(const WaveQ<C>& s, const f32x16_t (&acc)[C::MT], float (&out)[C::NIH]) {
  if constexpr (C::GROUPED) {
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int sq = 0; sq < C::GPQ; ++sq) {
          float sum = 0.0f;
#pragma unroll
          for (int r = 0; r < C::H; ++r) {
            const int v = 4 * i + sq * C::H + r;
            if constexpr (C::UNITW) sum = acc[mt][v];
            else sum = fmaf(s.wv[mt][v], relu<C>(acc[mt][v]), sum);
          }
          out[(mt * 4 + i) * C::GPQ + sq] = sum;
        }
  } else {
#pragma unroll
    for (int q = 0; q < C::QW; ++q) out[q] = 0.0f;
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int q = (32 * mt + 8 * i) / C::H;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int v = 4 * i + r;
          out[q] = fmaf(s.wv[mt][v], relu<C>(acc[mt][v]), out[q]);
        }
      }
  }
}

// Both sub-tiles' results -> the lane's NI complete scores. For H >= 8 the
// lane halves hold disjoint head subsets of the same (query, key): half 0
// finishes sub-tile 0 of query q, half 1 sub-tile 1, each sending the partial
// the other half needs.
template <class C>
__device__ __forceinline__ void combine(const float (&h0)[C::NIH], const float (&h1)[C::NIH], float (&sc)[C::NI]) {
  const int h = lane_id() >> 5;
  if constexpr (C::GROUPED) {
#pragma unroll
    for (int j = 0; j < C::NIH; ++j) {
      sc[j] = h0[j];
      sc[C::NIH + j] = h1[j];
    }
  } else {
#pragma unroll
    for (int it = 0; it < C::NI; ++it) {
      // v_permlane32_swap(x, y) exchanges x's upper 32 lanes with y's lower
      // 32 lanes: lanes 0-31 receive h0 of lane + 32 in y, lanes 32-63
      // receive h1 of lane - 32 in x.
      const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(h0[it]), __float_as_uint(h1[it]), false, false);
      sc[it] = h ? h1[it] + __uint_as_float(r[0]) : h0[it] + __uint_as_float(r[1]);
    }
  }
}

// Instruction pattern of one half step: per K slice, MFMA / 4 VALU / MFMA /
// 4 VALU / one LDS read of the next sub-tile's B fragment (issued as soon as
// the slice's fragment register is free), so the matrix pipe always has an
// MFMA queued and the epilogue of the other sub-tile runs in its shadow.
template <class C>
__device__ __forceinline__ void schedule_half() {
  constexpr int kMfma = 0x008, kValu = 0x002, kDsRead = 0x100;
  constexpr int kReadsPerSlice = C::M::FB / 16 > 0 ? C::M::FB / 16 : 1;
#pragma unroll
  for (int ks = 0; ks < C::KS; ++ks) {
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt) {
      __builtin_amdgcn_sched_group_barrier(kMfma, 1, 0);
      __builtin_amdgcn_sched_group_barrier(kValu, C::VALU_PER_MFMA, 0);
    }
    __builtin_amdgcn_sched_group_barrier(kDsRead, kReadsPerSlice, 0);
  }
}

// Histogram increment in LDS, issued as plain ds_add_u32. Written as an
// opaque instruction so that the compiler does not make it wait for the key
// tiles still streaming into LDS (loads into LDS count on vmcnt, and the
// compiler cannot tell the histogram from the tile ring): LDS operations of
// one wave complete in order, so the wave's later histogram reads still see
// the increment, and no other wave reads this wave's histogram rows.
__device__ __forceinline__ void lds_add(uint32_t* p, uint32_t v) {
  const uint32_t a = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint32_t*)p;
  asm volatile("ds_add_u32 %0, %1" ::"v"(a), "v"(v) : "memory");
}
__device__ __forceinline__ void lds_inc(uint32_t* p) { lds_add(p, 1u); }

// The lane index, computed where it is used: paths taken on few tiles derive
// their per-lane addresses from it instead of keeping them live across the
// scan.
__device__ __forceinline__ int lane_here() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// The first 16 bytes of a per-query LDS record and a slot from the query's
// LDS counter (ds_add_rtn_u32 of 1), issued together under one wait. Opaque
// for the same reason as lds_inc.
typedef float f32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint32_t lds_state_slot(const void* rec, uint32_t* ctr, f32x4_t& f) {
  const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)rec;
  const uint32_t b = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint32_t*)ctr;
  uint32_t r;
  asm volatile("ds_read_b128 %0, %2\n\tds_add_rtn_u32 %1, %3, %4\n\ts_waitcnt lgkmcnt(0)"
               : "=&v"(f), "=&v"(r)
               : "v"(a), "v"(b), "v"(1u)
               : "memory");
  return r;
}

// A slot from an LDS counter (ds_add_rtn_u32 of 1, the old value), LDS
// writes and reads, and a 32-byte per-query record read (as two 16-byte
// halves). Opaque for the same reason as lds_inc; the reads wait for their
// data.
__device__ __forceinline__ uint32_t lds_slot(uint32_t* ctr) {
  const uint32_t b = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint32_t*)ctr;
  uint32_t r;
  asm volatile("ds_add_rtn_u32 %0, %1, %2\n\ts_waitcnt lgkmcnt(0)" : "=v"(r) : "v"(b), "v"(1u) : "memory");
  return r;
}
__device__ __forceinline__ void lds_put4(float* p, f32x4_t v) {
  const uint32_t a = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) float*)p;
  asm volatile("ds_write_b128 %0, %1" ::"v"(a), "v"(v) : "memory");
}
__device__ __forceinline__ void lds_put1(uint32_t* p, uint32_t v) {
  const uint32_t a = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint32_t*)p;
  asm volatile("ds_write_b32 %0, %1" ::"v"(a), "v"(v) : "memory");
}
__device__ __forceinline__ uint32_t lds_get1(const uint32_t* p) {
  const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint32_t*)p;
  uint32_t r;
  asm volatile("ds_read_b32 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(r) : "v"(a) : "memory");
  return r;
}
// N (2 or 8) consecutive 16-byte LDS reads under one wait
template <int N>
__device__ __forceinline__ void lds_get_n(const float* p, f32x4_t (&o)[N]) {
  static_assert(N == 2 || N == 8, "record sizes of the grouped layouts");
  const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) float*)p;
  if constexpr (N == 2) {
    asm volatile("ds_read_b128 %0, %2\n\tds_read_b128 %1, %2 offset:16\n\ts_waitcnt lgkmcnt(0)"
                 : "=&v"(o[0]), "=&v"(o[1])
                 : "v"(a)
                 : "memory");
  } else {
    asm volatile(
        "ds_read_b128 %0, %8\n\tds_read_b128 %1, %8 offset:16\n\t"
        "ds_read_b128 %2, %8 offset:32\n\tds_read_b128 %3, %8 offset:48\n\t"
        "ds_read_b128 %4, %8 offset:64\n\tds_read_b128 %5, %8 offset:80\n\t"
        "ds_read_b128 %6, %8 offset:96\n\tds_read_b128 %7, %8 offset:112\n\ts_waitcnt lgkmcnt(0)"
        : "=&v"(o[0]), "=&v"(o[1]), "=&v"(o[2]), "=&v"(o[3]), "=&v"(o[4]), "=&v"(o[5]), "=&v"(o[6]), "=&v"(o[7])
        : "v"(a)
        : "memory");
  }
}
__device__ __forceinline__ void lds_get_rec(const void* rec, f32x4_t& f, i32x4_t& g) {
  const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)rec;
  asm volatile("ds_read_b128 %0, %2\n\tds_read_b128 %1, %2 offset:16\n\ts_waitcnt lgkmcnt(0)"
               : "=&v"(f), "=&v"(g)
               : "v"(a)
               : "memory");
}

// (v << 1) | !(a < b): the compare writes VCC, the add with carry doubles v
// and adds the carry.
__device__ __forceinline__ uint32_t shift_in_nlt(uint32_t v, float a, float b) {
  uint32_t r;
  asm("v_cmp_nlt_f32 vcc, %1, %2\n\tv_addc_co_u32 %0, vcc, %3, %3, vcc" : "=v"(r) : "v"(a), "v"(b), "v"(v) : "vcc");
  return r;
}

// Key sources: consecutive positions (kContig, staged through a buffer
// descriptor per tile) or a list of key indices (gathered per row).
struct SrcContig {
  static constexpr bool kContig = true;
  __device__ int key(int i) const { return i; }
};
template <bool FAR>
struct SrcListT {
  static constexpr bool kContig = false;
  static constexpr bool kFar = FAR;  // keys beyond 4 GiB: per-lane global addresses
  const int32_t* list;
  __device__ int raw(int i) const { return list[i]; }
  // a list entry as a key index (hole markers -1 read key 0; never used)
  __device__ static int clamp(int v) { return v < 0 ? 0 : v; }
  __device__ int key(int i) const { return clamp(raw(i)); }
};
using SrcList = SrcListT<false>;
using SrcListFar = SrcListT<true>;

// The block-wide scan of positions [kbeg, kend) of `src` (key index =
// src.key(position)). Keys flow HBM -> LDS through a ring of four tiles
// (loads three tiles ahead, one barrier per tile). Each tile is processed in
// two half steps that overlap the matrix cores with the vector ALUs: while
// the MFMAs of one 32-key sub-tile run, the epilogue of the other sub-tile
// (and the sink's gate / write-back for the previous tile) executes. B
// fragments are read from LDS one half step ahead. The loop is unrolled over
// the ring, so every LDS address of a B fragment is a per-lane register plus
// an immediate.
template <class C, class Src, class Sink>
__device__ __forceinline__ void wg_scan(const ScoreArgs& a, const Src& src, int kbeg, int kend, uint8_t* tiles,
                                        const WaveQ<C>& wq, Sink& sink) {
  using Frag = typename C::M::Frag;
  const int tid = threadIdx.x, l = lane_id(), h = l >> 5, r32 = l & 31;
  const uint8_t* keys = static_cast<const uint8_t*>(a.keys);
  // the bounds are the same in every lane; saying so keeps the per-tile
  // descriptors below in scalar registers
  kbeg = __builtin_amdgcn_readfirstlane(kbeg);
  kend = __builtin_amdgcn_readfirstlane(kend);
  const int nsteps = kend > kbeg ? (kend - kbeg + C::KT - 1) / C::KT : 0;
  if (nsteps == 0) return;
  // Key tiles go straight from HBM to LDS (loads into LDS, 16 bytes per
  // lane): each instruction of a wave fills 64 consecutive 16-byte chunk
  // slots. A contiguous source loads through a buffer descriptor based at the
  // tile's first key and sized to the keys left before kend: each lane's
  // offset is fixed for the whole scan, and rows past kend fall outside the
  // descriptor (their slots hold whatever the hardware returns; every
  // consumer masks positions >= kend). A list source gathers its rows, past
  // kend clamped to the last valid position.
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  uint32_t voff[C::CPT];
#pragma unroll
  for (int c = 0; c < C::CPT; ++c) {
    const int u = (c * C::WAVES + wave) * kWave + l, n = u / C::CPK, part = (u ^ C::swz(n)) & (C::CPK - 1);
    voff[c] = (uint32_t)(n * C::ROWB + part * 16);
  }
  // A list source's key indices for the next tile to stage, read one tile
  // ahead: a list read that the stage itself waited on would also wait for
  // every tile load in flight (vector-memory loads complete in issue order).
  int lk[C::CPT], lks = 0;
  auto list_keys = [&](int k0) {
    if constexpr (!Src::kContig) {
#pragma unroll
      for (int c = 0; c < C::CPT; ++c) {
        const int u = (c * C::WAVES + wave) * kWave + l, n = u / C::CPK;
        lk[c] = src.raw(min(k0 + n, kend - 1));
      }
      if constexpr (C::DT == DT_FP8) lks = src.raw(min(k0 + l, kend - 1));
    }
  };
  list_keys(kbeg);
  auto stage = [&](int slot, int st_abs, int k0) {
    if constexpr (Src::kContig) {
      // rows of this tile before kend, kept in a scalar register (a vector
      // clamp would make the descriptor look different per lane)
      int rows = kend - k0;
      asm volatile("" : "+s"(rows));
      rows = rows < 0 ? 0 : rows;
      asm volatile("" : "+s"(rows));
      rows = rows > C::KT ? C::KT : rows;
      if constexpr (C::DT == DT_FP8) {
        // wave 0 copies the tile's key scales (64 lanes x 4 bytes) ahead of
        // its key chunks, so the key chunks stay the newest loads in flight
        if (wave == 0) {
          uint8_t* d = tiles + C::RING * C::TILE_BYTES + (st_abs & (C::SCALE_RING - 1)) * C::KT * 4;
          const __amdgpu_buffer_rsrc_t rs =
              __builtin_amdgcn_make_buffer_rsrc((void*)(a.k_scale + k0), 0, rows * 4, kBufferRaw);
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (void __attribute__((address_space(3)))*)d, 4,
                                                   (uint32_t)l * 4u, 0, 0, 0);
        }
      }
      const __amdgpu_buffer_rsrc_t rs =
          __builtin_amdgcn_make_buffer_rsrc((void*)(keys + (int64_t)k0 * C::ROWB), 0, rows * C::ROWB, kBufferRaw);
#pragma unroll
      for (int c = 0; c < C::CPT; ++c) {
        uint8_t* d = tiles + slot * C::TILE_BYTES + (c * C::WAVES + wave) * kWave * 16;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (void __attribute__((address_space(3)))*)d, 16, voff[c], 0, 0,
                                                 0);
      }
    } else {
      // addresses from the keys read one tile ago; then the next tile's keys,
      // issued ahead of this tile's loads so that the tile wait covers them
      const uint32_t soff = (uint32_t)Src::clamp(lks);
      const float* gs = a.k_scale + soff;
      const uint8_t* g[C::CPT];
#pragma unroll
      for (int c = 0; c < C::CPT; ++c) {
        const int u = (c * C::WAVES + wave) * kWave + l, n = u / C::CPK, part = (u ^ C::swz(n)) & (C::CPK - 1);
        g[c] = keys + (int64_t)Src::clamp(lk[c]) * C::ROWB + part * 16;
      }
      list_keys(k0 + C::KT);
      asm volatile("" ::: "memory");
      if constexpr (!Src::kFar) {
        // keys within 4 GiB: byte offsets from the array's start through a
        // buffer descriptor (loads into LDS through a descriptor keep the
        // compiler's LDS waits exact; see the contiguous case)
        if constexpr (C::DT == DT_FP8) {
          if (wave == 0) {
            uint8_t* d = tiles + C::RING * C::TILE_BYTES + (st_abs & (C::SCALE_RING - 1)) * C::KT * 4;
            const __amdgpu_buffer_rsrc_t rs =
                __builtin_amdgcn_make_buffer_rsrc((void*)a.k_scale, 0, a.nk * 4, kBufferRaw);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (void __attribute__((address_space(3)))*)d, 4,
                                                     soff * 4u, 0, 0, 0);
          }
        }
        const __amdgpu_buffer_rsrc_t rs =
            __builtin_amdgcn_make_buffer_rsrc((void*)keys, 0, (int)((uint32_t)a.nk * (uint32_t)C::ROWB), kBufferRaw);
#pragma unroll
        for (int c = 0; c < C::CPT; ++c) {
          uint8_t* d = tiles + slot * C::TILE_BYTES + (c * C::WAVES + wave) * kWave * 16;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (void __attribute__((address_space(3)))*)d, 16,
                                                   (uint32_t)(g[c] - keys), 0, 0, 0);
        }
      } else {
        if constexpr (C::DT == DT_FP8) {
          if (wave == 0) {
            uint8_t* d = tiles + C::RING * C::TILE_BYTES + (st_abs & (C::SCALE_RING - 1)) * C::KT * 4;
            __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)gs,
                                             (void __attribute__((address_space(3)))*)d, 4, 0, 0);
          }
        }
#pragma unroll
        for (int c = 0; c < C::CPT; ++c) {
          uint8_t* d = tiles + slot * C::TILE_BYTES + (c * C::WAVES + wave) * kWave * 16;
          __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)g[c],
                                           (void __attribute__((address_space(3)))*)d, 16, 0, 0);
        }
      }
    }
  };
  // Wait until at most `n` of this wave's vector-memory operations are in
  // flight (loads complete in issue order), then a plain barrier: the tile
  // whose loads are done is visible to every wave. No release fence -- it
  // would wait for every outstanding load, including the prefetches.
  auto sync_tiles = [&](int n) {
    asm volatile("" ::: "memory");
    if (n == 0) __builtin_amdgcn_s_waitcnt(0x0F70);
    else __builtin_amdgcn_s_waitcnt(0x0F70 | C::CPT);
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };
  // both sub-tiles' results of tile st -> complete scores (fp8: key scales)
  auto scores = [&](int st, const float (&h0)[C::NIH], const float (&h1)[C::NIH], float (&sc)[C::NI]) {
    combine<C>(h0, h1, sc);
    if constexpr (C::DT == DT_FP8) {
#pragma unroll
      for (int it = 0; it < C::NI; ++it) {
        const int nt = h ? C::item_nt(it, 1) : C::item_nt(it, 0);
        const float* sl = reinterpret_cast<const float*>(tiles + C::RING * C::TILE_BYTES) +
                          (st & (C::SCALE_RING - 1)) * C::KT;
        sc[it] *= sl[nt * 32 + r32];
      }
    }
  };

  stage(0, 0, kbeg);
  stage(1, 1, kbeg + C::KT);
  stage(2, 2, kbeg + 2 * C::KT);
  sync_tiles(1);  // tiles 0 and 1 landed (tile 2 may still be in flight)
  Frag b0[C::KS], b1[C::KS];
  f32x16_t acc0[C::MT], acc1[C::MT];
#pragma unroll
  for (int mt = 0; mt < C::MT; ++mt) acc1[mt] = f32x16_t{};
  float h0[C::NIH], h1[C::NIH];
#pragma unroll
  for (int j = 0; j < C::NIH; ++j) h0[j] = 0.0f;
  BLane<C> bl;
  bl.init(tiles);
  load_b_at<C, 0, 0>(tiles, bl, b0);
  // one tile; SLOT = st % RING, a constant in every copy of the body
  static_assert(C::RING == 4, "the loop is unrolled over the ring");
  auto body = [&](auto SLOT_, int st) {
    constexpr int SLOT = decltype(SLOT_)::value;
    bl.opaque();
    // the sink's loads for this step go ahead of the tile loads, so that the
    // step's tile wait covers them
    if constexpr (requires { sink.pre(); }) sink.pre();
    // slot of tile st-1 is free: every wave passed the barrier after reading it
    stage((SLOT + 3) & 3, st + 3, kbeg + (st + 3) * C::KT);
    // half step A: MFMA sub-tile 0 of tile st || epilogue of sub-tile 1 of st-1,
    // B fragments of sub-tile 1 read as the slots free up
    mma_half<C>(wq, b0, acc0);
    load_b_at<C, SLOT, 1>(tiles, bl, b1);
    reduce_half<C>(wq, acc1, h1);
    float sc[C::NI];
    scores(st - 1, h0, h1, sc);
    schedule_half<C>();
    // half step B: MFMA sub-tile 1 of tile st || epilogue of sub-tile 0 of st,
    // B fragments of the next tile's sub-tile 0 read as the slots free up
    mma_half<C>(wq, b1, acc1);
    load_b_at<C, (SLOT + 1) & 3, 0>(tiles, bl, b0);
    reduce_half<C>(wq, acc0, h0);
    schedule_half<C>();
    // h0 is only read in the next step; without this use the compiler sinks
    // its epilogue below the gate's branches, out of the MFMA shadow
#pragma unroll
    for (int j = 0; j < C::NIH; ++j) asm volatile("" ::"v"(h0[j]));
    // gate + write-back of tile st-1 while the last MFMAs drain
    sink.consume(st - 1, kbeg + (st - 1) * C::KT, kend, sc, st > 0);
    sync_tiles(1);  // tile st+2 landed; tile st+3 may still be in flight
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
  int st = 0;
  for (; st + C::RING <= nsteps; st += C::RING) {
    body(I0{}, st);
    body(I1{}, st + 1);
    body(I2{}, st + 2);
    body(I3{}, st + 3);
  }
  if (st < nsteps) body(I0{}, st++);
  if (st < nsteps) body(I1{}, st++);
  if (st < nsteps) body(I2{}, st++);
  reduce_half<C>(wq, acc1, h1);
  float sc[C::NI];
  scores(nsteps - 1, h0, h1, sc);
  sink.consume(nsteps - 1, kbeg + (nsteps - 1) * C::KT, kend, sc, true);
  sync_tiles(0);  // no prefetch may still be writing LDS when the caller reuses it
}

// ---------------------------------------------------------------------------
// Sinks. consume(st, k0, kend, scores, live) receives the scores of tile st
// (positions k0 + ...); live is false for the pipeline's priming call.
// ---------------------------------------------------------------------------

// Writes every score to out[t * ld + position].
template <class C>
struct DenseSink {
  float* out;
  int64_t ld;
  int qbase, nq;
  __device__ void consume(int, int k0, int kend, const float (&sc)[C::NI], bool live) {
    const int l = lane_id(), h = l >> 5, r32 = l & 31;
#pragma unroll
    for (int it = 0; it < C::NI; ++it) {
      const int q = h ? C::item_q(it, 1) : C::item_q(it, 0);
      const int nt = h ? C::item_nt(it, 1) : C::item_nt(it, 0);
      const int pos = k0 + nt * 32 + r32, t = qbase + q;
      if (live && t < nq && pos < kend) out[(int64_t)t * ld + pos] = sc[it];
    }
  }
};

// Writes the scores of the fallback's batch of rows: query t of the block's
// tile goes to out[slot * ld + position] when slot = smap[t - q0] >= 0 (the
// map is in LDS, [QT] entries).
template <class C>
struct RowSink {
  float* out;
  int64_t ld;
  const int8_t* smap;
  int qbase, q0;
  __device__ void consume(int, int k0, int kend, const float (&sc)[C::NI], bool live) {
    const int l = lane_id(), h = l >> 5, r32 = l & 31;
#pragma unroll
    for (int it = 0; it < C::NI; ++it) {
      const int q = h ? C::item_q(it, 1) : C::item_q(it, 0);
      const int nt = h ? C::item_nt(it, 1) : C::item_nt(it, 0);
      const int pos = k0 + nt * 32 + r32;
      const int slot = smap[qbase + q - q0];
      if (live && slot >= 0 && pos < kend) out[slot * ld + pos] = sc[it];
    }
  }
};

// The fused filter (sec. 3.2 "Filtering" and "Threshold Refresh") for the
// wave's QW rows. Per score: bin-space value x = fma(I, delta, c), gate
// !(x < thr) with thr the current threshold bin, causal mask. Passing scores
// are compacted with one ballot per item (mbcnt gives each passing lane its
// slot; the row's tail is wave-private, so no atomics), written as (key,
// score) to the row's HBM candidate list, and counted in the row's LDS
// histogram.
// Threshold refresh: the wave keeps, per row, `above` = the number of counted
// candidates in bins strictly above the current threshold bin tau. Whenever
// above >= k, bin tau + 1 still has a suffix count >= k, so tau advances and
// above drops by the count of the bin it moves to. This keeps tau equal to
// the histogram walk's result (the largest bin whose suffix count reaches k)
// after every tile, at the cost of one ballot per item and a short loop only
// when the threshold actually moves.
template <class C>
struct FusedSink {
  float delta[C::QW], cc[C::QW], thr[C::QW], thr_up[C::QW];
  int tau[C::QW], e[C::QW], sv[C::QW];
  uint32_t tail[C::QW], above[C::QW];
  uint32_t* hist;     // LDS, [QW][m] for this wave
  int2* cand;
  int2* crow[C::QW];  // this split's candidate list of each query
  const int32_t* rflag;  // second filter pass: only rows with rflag[t] set (else NULL: every row)
  int qbase, nq, S, split, cap, m, k;

  __device__ __forceinline__ bool row_on(int t) const { return t < nq && (!rflag || rflag[t]); }

  __device__ __forceinline__ void set_tau(int q, int t) {
    tau[q] = t;
    thr[q] = gate_thr(t);
    thr_up[q] = t < m - 1 ? (float)(t + 1) : __builtin_nanf("");
  }

  __device__ __forceinline__ void init(const ScoreArgs& a, const RowParam* params, int kend) {
#pragma unroll
    for (int q = 0; q < C::QW; ++q) {
      const int t = qbase + q;
      RowRange rr{0, 0};
      float dl = 1.0f, c = 0.0f;
      int t0 = -1;
      if (row_on(t)) {
        rr = row_range(a.offs, a.starts, t, a.nk);
        const RowParam p = params[t];
        dl = p.delta;
        c = p.c;
        t0 = p.tau0;
      }
      e[q] = rr.e < kend ? rr.e : kend;
      sv[q] = rr.s;
      crow[q] = cand + ((int64_t)(t < nq ? t : 0) * S + split) * cap;
      delta[q] = dl;
      cc[q] = c;
      set_tau(q, t0);
      tail[q] = 0;
      above[q] = 0;
    }
  }

  __device__ __forceinline__ void consume(int, int k0, int, const float (&sc)[C::NI], bool live) {
    const int l = lane_id(), h = l >> 5, r32 = l & 31;
    float x[C::NI];
    bool ps[C::NI];
    uint64_t any = 0;
    static_for<C::NI>([&](auto IT) {
      constexpr int it = decltype(IT)::value;
      constexpr int qa = C::item_q(it, 0), qb = C::item_q(it, 1);
      constexpr int na = C::item_nt(it, 0), nb = C::item_nt(it, 1);
      const int key = k0 + (h ? nb : na) * 32 + r32;
      x[it] = bin_x(sc[it], h ? delta[qb] : delta[qa], h ? cc[qb] : cc[qa]);
      ps[it] = live && key < (h ? e[qb] : e[qa]) && key >= (h ? sv[qb] : sv[qa]) &&
               !(x[it] < (h ? thr[qb] : thr[qa]));
      any |= __ballot(ps[it]);
    });
    if (any == 0) return;  // wave-uniform: nothing passed this tile
    static_for<C::NI>([&](auto IT) {
      constexpr int it = decltype(IT)::value;
      constexpr int qa = C::item_q(it, 0), qb = C::item_q(it, 1);
      constexpr int na = C::item_nt(it, 0), nb = C::item_nt(it, 1);
      const bool pass = ps[it];
      const uint64_t mask = __ballot(pass);
      const uint64_t up = __ballot(pass && x[it] >= (h ? thr_up[qb] : thr_up[qa]));
      const uint32_t mb = mbcnt64(mask);
      uint32_t pos;
      if constexpr (qa == qb) {
        pos = tail[qa] + mb;
        tail[qa] += (uint32_t)__popcll(mask);
        above[qa] += (uint32_t)__popcll(up);
      } else {
        const uint32_t lo = (uint32_t)__popcll(mask & 0xFFFFFFFFull);
        pos = h ? tail[qb] + mb - lo : tail[qa] + mb;
        tail[qa] += lo;
        tail[qb] += (uint32_t)__popcll(mask) - lo;
        const uint32_t ulo = (uint32_t)__popcll(up & 0xFFFFFFFFull);
        above[qa] += ulo;
        above[qb] += (uint32_t)__popcll(up) - ulo;
      }
      if (pass) {
        const int key = k0 + (h ? nb : na) * 32 + r32;
        const int q = h ? qb : qa;
        if (pos < (uint32_t)cap) crow[q][pos] = make_int2(key, __float_as_int(sc[it]));
        // bin_of without branches: x >= 0 excludes NaN and the below-range scores
        const float xv = x[it];
        if (xv >= 0.0f) lds_inc(&hist[q * m + min(__float2int_rz(xv), m - 1)]);
      }
    });
#pragma unroll
    for (int q = 0; q < C::QW; ++q) {
      if (above[q] >= (uint32_t)k) {
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        int t = tau[q];
        uint32_t ab = above[q];
        while (ab >= (uint32_t)k && t < m - 1) {
          ++t;
          ab -= hist[q * m + t];
        }
        above[q] = ab;
        set_tau(q, t);
      }
    }
  }

  __device__ __forceinline__ void finish(uint32_t* cnt, uint32_t* hist_out) {
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    const int l = lane_id();
#pragma unroll
    for (int q = 0; q < C::QW; ++q) {
      const int t = qbase + q;
      if (!row_on(t)) continue;
      const int64_t u = (int64_t)t * S + split;
      for (int b = l; b < m; b += kWave) hist_out[u * m + b] = hist[q * m + b];
      if (l == 0) cnt[u] = tail[q];
    }
  }
};

// The fused filter for layouts where a lane holds whole scores of many queries
// (H <= 4: up to 32 queries per wave, 32 scores per lane per tile, e.g. the
// one-head inner-product retrieval scorer). The per-query state (visible
// range, bin map, thresholds, list length, counts above the thresholds) lives
// in LDS, one 32-byte record per query plus three counters, so that a lane
// reaches the state of whichever query its score belongs to with one gather,
// and list slots and counts are taken with LDS atomics by every passing lane
// at once.
// Gate in the score domain: bin(fma(I, delta, c)) >= tau holds for every
// I >= (tau - c) / delta (real division; fma rounding is monotone and tau is
// a float), so the lane compares each score with T, that quotient lowered by
// far more than its float rounding error: one compare per score, never
// dropping a key whose bin is >= tau. A key let through just below the bin
// edge is written and counted in its true (lower) bin, which changes neither
// the refresh (it only reads bins above tau) nor the final select (it keeps
// bins >= the final threshold, whose counts stay complete). Scores that pass
// the compare are re-checked against the visible range of their row before
// they are written. NaN passes the compare (as in the bin gate) and is never
// counted. The order of a list's entries depends on the order in which the
// atomics are served; the final select orders candidates by (score, key)
// alone, so no result depends on it.
// Passing scores are not written out in the tile that finds them: every
// lane with one appends a record of its tile scores to the wave's LDS queue
// (a ballot, mbcnt for the slot, a few LDS writes, no round trip), and every
// kDrainEvery tiles all waves drain their queues at once, one record per
// lane, re-checking each score against its row's current gate.
// Handled where found, the per-item work of one wave held up the other waves
// of its block at the tile barrier on most tiles; drained together, no wave
// waits for another, and the counting's LDS round trips serve many records
// at a time. The thresholds then move up to kDrainEvery tiles later, which
// only lets a few more keys through. A tile with more passing lanes than the
// queue holds (a row without a gate) is handled in place.
// Key splits of one row share a threshold (2 to 8 splits; every kShareEvery
// tiles a wave reads its rows' published bins). Besides its own bin tau
// (the largest bin with at least k of the split's candidates at or above
// it), each split tracks tau_s, the same walk for ks = ceil(k / S), and
// publishes it in its byte of the row's entry in `pub`. The smallest bin g
// the S splits of a row have published has at least ks candidates of every
// split at or above it, S * ks >= k keys of the row in all, so g never
// exceeds the row's final threshold bin over all splits; every split raises
// its own bin to g. (Sharing the largest own bin instead would keep each
// split at its own top k; the smallest of the ks walks follows the top k of
// all splits together.) A raised gate drops only keys below the final bin,
// and the counts at and above that bin stay complete in every histogram.
template <class C>
struct GroupedSink {
  static_assert(C::GROUPED && C::QW <= kWave, "one query per lane");
  // LDS record of one query: the first 16 bytes are what a passing score
  // needs (bin map and the bins above the two thresholds), the rest what the
  // threshold updates and the range check read
  struct alignas(16) QState {
    float delta, c;  // bin-space value x = fma(I, delta, c)
    float up;        // (float)(tau + 1): x >= up is a count above tau; +inf at the top bin
    float ups;       // the same for tau_s
    float gate;      // T, the score-domain gate (+inf for rows past the end)
    int s, e;        // visible keys [s, e) within this split
    int pad;
  };
  static constexpr int kRecs = 32;        // records of a wave's queue: a lane's scores of one tile
  static constexpr int kDrainEvery = 16;  // tiles between queue drains
  static constexpr int kShareEvery = 8;   // tiles between reads of the published bins
  static constexpr int kLdsPerWave =
      C::QW * (int)sizeof(QState) + 3 * C::QW * 4 + kRecs * C::NI * 4 + ((kRecs * 4 + 15) & ~15);
  static_assert(C::NI % 4 == 0 && (C::QW * 12) % 16 == 0, "16-byte aligned records");
  QState* qs;         // LDS [QW]
  uint32_t* tail;     // LDS [QW]: candidates passed (the list length; may exceed cap)
  uint32_t* above;    // LDS [QW]: counted candidates in bins above tau
  uint32_t* above_s;  // LDS [QW]: the same above tau_s
  float* rec;         // LDS [kRecs][NI]: a lane's scores of one tile
  uint32_t* rhdr;     // LDS [kRecs]: (tile's first key - kq0) << 8 | lane
  int qlen;           // records in the queue
  int kq0;            // first key of the split
  bool use_queue;     // keys of the split are told apart by 24 bits
  float tq[C::NIH];   // T of the query of item j (items j and j + NIH share it)
  bool ungated;       // some row of the wave has no gate (tau = -1)
  int vis_s, vis_e;   // every row of the wave sees [vis_s, vis_e)
  uint8_t* pub;       // [nq][8] published bins + 1 of the row's splits (2 to 8), or NULL
  int tau_v, taus_v;  // lane q: tau and tau_s of query qbase + q
  uint64_t gw;        // lane q: its row's published bytes, as read
  int ks, steps, ntile;
  uint32_t* hist;     // LDS, [QW][m] for this wave
  int2* cand;
  int64_t lbase, lstride;  // list of query q: cand + lbase + q * lstride
  const int32_t* rflag;    // second filter pass: only rows with rflag[t] set (else NULL: every row)
  int qbase, nq, S, split, cap, m, k;

  __device__ __forceinline__ bool row_on(int t) const { return t < nq && (!rflag || rflag[t]); }

  __device__ __forceinline__ void bind(uint8_t* lds) {
    qs = reinterpret_cast<QState*>(lds);
    tail = reinterpret_cast<uint32_t*>(lds + C::QW * sizeof(QState));
    above = tail + C::QW;
    above_s = above + C::QW;
    rec = reinterpret_cast<float*>(above_s + C::QW);
    rhdr = reinterpret_cast<uint32_t*>(rec + kRecs * C::NI);
  }

  __device__ __forceinline__ static float gate_floor(float delta, float c, int tau) {
    if (tau < 0) return -__builtin_inff();
    const float t = (float)tau, i0 = (t - c) / delta;
    const float err = ((fabsf(t) + fabsf(c)) / delta + fabsf(i0)) * 0x1p-20f;
    return i0 - err;
  }

  __device__ __forceinline__ float up_of(int t) const { return t < m - 1 ? (float)(t + 1) : __builtin_inff(); }

  // the per-item copies of T, and the ungated flag (the query of item j in
  // lane half h is item_q(j, 0) + h * 4 / H)
  __device__ __forceinline__ void update_gates() {
    const int l = lane_here();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    const QState* qh = qs + (l >> 5) * (4 / C::H);
    static_for<C::NIH>([&](auto J) {
      constexpr int j = decltype(J)::value;
      static_assert(C::item_q(j, 1) - C::item_q(j, 0) == 4 / C::H, "query of an item in the upper half");
      tq[j] = qh[C::item_q(j, 0)].gate;
    });
    const bool valid = l < C::QW && row_on(qbase + l);
    ungated = __ballot(valid && tau_v < 0) != 0;
  }

  __device__ __forceinline__ void init(const ScoreArgs& a, const RowParam* params, int kend) {
    const int l = lane_id(), t = qbase + l;
    const bool valid = l < C::QW && row_on(t);
    RowRange rr{0, 0};
    float dl = 1.0f, c = 0.0f;
    int t0 = -1;
    if (valid) {
      rr = row_range(a.offs, a.starts, t, a.nk);
      const RowParam p = params[t];
      dl = p.delta;
      c = p.c;
      t0 = p.tau0;
    }
    const int e = rr.e < kend ? rr.e : kend;
    // the wave's common range (empty rows past the end do not narrow it)
    int cs = valid ? rr.s : 0, ce = valid ? e : INT_MAX;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      cs = max(cs, __shfl_xor(cs, o));
      ce = min(ce, __shfl_xor(ce, o));
    }
    vis_s = __builtin_amdgcn_readfirstlane(cs);
    vis_e = __builtin_amdgcn_readfirstlane(ce);
    lstride = (int64_t)S * cap;
    lbase = ((int64_t)qbase * S + split) * cap;
    ks = (k + S - 1) / S;
    steps = 0;
    ntile = 0;
    qlen = 0;
    // tiles start at kq0 + 64 j, so the last one ends below kq0 + 2^24
    use_queue = kend - kq0 < (1 << 24);
    tau_v = valid ? t0 : m - 1;
    taus_v = tau_v;
    gw = 0;
    if (l < C::QW) {
      QState r;
      r.delta = dl;
      r.c = c;
      r.up = up_of(tau_v);
      r.ups = r.up;
      r.gate = valid ? gate_floor(dl, c, t0) : __builtin_inff();
      r.s = rr.s;
      r.e = e;
      r.pad = 0;
      qs[l] = r;
      tail[l] = 0u;
      above[l] = 0u;
      above_s[l] = 0u;
    }
    update_gates();
  }

  // every kShareEvery steps: read the rows' published bins (lands by the
  // step's tile wait)
  __device__ __forceinline__ void pre() {
    if (!pub) return;
    if (steps++ % kShareEvery != 0) return;
    const int l = lane_id();
    if (l < C::QW && qbase + l < nq)
      gw = __hip_atomic_load(reinterpret_cast<uint64_t*>(pub) + qbase + l, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
  }

  // lane lq: its query's bin moves to t (above already adjusted)
  __device__ __forceinline__ void move_tau(int lq, int t, uint32_t ab) {
    above[lq] = ab;
    QState& r = qs[lq];
    r.up = up_of(t);
    r.gate = gate_floor(r.delta, r.c, t);
    tau_v = t;
  }

  __device__ __forceinline__ void consume(int, int k0, int, const float (&sc)[C::NI], bool live) {
    if (!live) return;
    static_assert(C::NI <= 32, "one bit per item");
    typedef float fNI __attribute__((ext_vector_type(C::NI)));
    const int l = lane_id(), h = l >> 5, r32 = l & 31;
    // raise each row's bin to the smallest bin its splits have published
    if (pub && (steps - 1) % kShareEvery == 0) {
      int g = 255;
      for (int j = 0; j < S; ++j) g = min(g, (int)((gw >> (8 * j)) & 0xFFu));
      g -= 1;
      const bool raise = l < C::QW && row_on(qbase + l) && g > tau_v;
      if (__ballot(raise) != 0) {
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        if (raise) {
          const int lq = lane_here();
          uint32_t ab = above[lq];
          for (int t = tau_v + 1; t <= g; ++t) ab -= hist[lq * m + t];
          move_tau(lq, g, ab);
        }
        update_gates();
      }
    }
    // the periodic drain, at the same tile in every wave
    if (use_queue && ++ntile % kDrainEvery == 0 && qlen != 0) {
      drain();
      refresh();
    }
    // fast path, vector ALU only (a chain of per-item ballots would stall on
    // every scalar read of a compare result): the largest margin score - T
    // over the lane's items; T - T' < 0 for every non-NaN score below its T.
    // A NaN score only matters to an ungated row, and then the fast path is
    // skipped.
    static_assert(C::NI == 2 * C::NIH, "items j and j + NIH share their query");
    if (!ungated) {
      float mx = -__builtin_inff();
#pragma unroll
      for (int j = 0; j < C::NIH; ++j) mx = fmaxf(mx, fmaxf(sc[j], sc[j + C::NIH]) - tq[j]);
      const bool lp = mx >= 0.0f;  // some score of this lane passes
      const uint64_t lm = __ballot(lp);
      if (lm == 0) return;  // wave-uniform: nothing passes
      if (use_queue) {
        // append a record of every such lane: its scores and where they are
        const int nrec = __popcll(lm);
        if (qlen + nrec > kRecs) {
          drain();
          refresh();
        }
        if (nrec <= kRecs) {
          if (lp) {
            const int slot = qlen + (int)mbcnt64(lm);
            float* rp = rec + slot * C::NI;
#pragma unroll
            for (int v = 0; v < C::NI / 4; ++v)
              lds_put4(rp + 4 * v, f32x4_t{sc[4 * v], sc[4 * v + 1], sc[4 * v + 2], sc[4 * v + 3]});
            lds_put1(rhdr + slot, (uint32_t)(k0 - kq0) << 8 | (uint32_t)l);
          }
          qlen += nrec;
          return;
        }
      }
    }
    // bit it of `bits`: this lane's score of item it passed the compare
    // (built from the top item down: a compare and a shift-add of its result)
    uint32_t bits = 0;
#pragma unroll
    for (int it = C::NI - 1; it >= 0; --it) bits = shift_in_nlt(bits, sc[it], tq[it % C::NIH]);
    const uint32_t items = wave_or(bits);
    if (items == 0) return;
    fNI scv;
#pragma unroll
    for (int it = 0; it < C::NI; ++it) scv[it] = sc[it];
    // in place, one item at a time: every passing lane takes its slot and
    // counts at once
    const bool inside = k0 >= vis_s && k0 + C::KT <= vis_e;
    for (uint32_t rem = items; rem; rem &= rem - 1) {
      const int it = __builtin_ctz(rem);
      if (!((bits >> it) & 1u)) continue;
      const int j = it % C::NIH, nt = it / C::NIH;
      const int q = item_query(j, h);
      const int key = k0 + nt * 32 + r32;
      if (!inside) {
        const QState& r = qs[q];
        if (key < r.s || key >= r.e) continue;
      }
      const float s_it = scv[it];
      f32x4_t f;
      const uint32_t pos = lds_state_slot(&qs[q], &tail[q], f);
      count(q, s_it, f);
      if (pos < (uint32_t)cap) cand[lbase + q * lstride + pos] = make_int2(key, __float_as_int(s_it));
    }
    refresh();
  }

  // counts of a written candidate of query q: its bin, and above tau / tau_s
  // (only when x >= 0: not NaN, not below the range; the adds are issued
  // either way, of 0 for the others, so that no branch is taken)
  __device__ __forceinline__ void count(int q, float s, const f32x4_t& f) {
    const float x = fmaf(s, f[0], f[1]);
    const int b = min(max(__float2int_rz(x), 0), m - 1);
    lds_add(&hist[q * m + b], x >= 0.0f ? 1u : 0u);
    lds_add(&above[q], x >= f[2] ? 1u : 0u);
    lds_add(&above_s[q], x >= f[3] ? 1u : 0u);
  }

  // the queue, one record per lane: the record's scores still at or above
  // their row's gate and inside its visible range take a slot, are written
  // and counted
  __device__ __forceinline__ void drain() {
    static_assert(kRecs <= kWave, "one record per lane");
    const int l = lane_here();
    if (l < qlen) {
      const float* rp = rec + l * C::NI;
      f32x4_t sv[C::NI / 4];
      lds_get_n<C::NI / 4>(rp, sv);
      const uint32_t hd = lds_get1(rhdr + l);
      const int src = (int)(hd & 0xFFu), hs = src >> 5, k0 = kq0 + (int)(hd >> 8);
      const int key0 = k0 + (src & 31);
      // the record's queries in its lane half: item_q(j, 0) + hs * 4 / H
      const QState* qh = qs + hs * (4 / C::H);
      uint32_t bits = 0;
#pragma unroll
      for (int it = C::NI - 1; it >= 0; --it)
        bits = shift_in_nlt(bits, sv[it / 4][it % 4], qh[C::item_q(it % C::NIH, 0)].gate);
      while (bits) {
        const int it = __builtin_ctz(bits);
        bits &= bits - 1;
        const int j = it % C::NIH, nt = it / C::NIH;
        const int q = item_query(j, hs);
        const int key = key0 + nt * 32;
        const float s = __uint_as_float(lds_get1(reinterpret_cast<const uint32_t*>(rp) + it));
        f32x4_t f;
        i32x4_t g;
        lds_get_rec(&qs[q], f, g);  // g: gate bits, s, e
        if (key >= g[1] && key < g[2]) {
          const uint32_t pos = lds_slot(&tail[q]);
          count(q, s, f);
          if (pos < (uint32_t)cap) cand[lbase + q * lstride + pos] = make_int2(key, __float_as_int(s));
        }
      }
    }
    qlen = 0;
  }

  // threshold refresh: each lane walks its own query's histogram, for tau
  // (k) and, where the splits share, for tau_s (ks)
  __device__ __forceinline__ void refresh() {
    const int l = lane_id();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    const bool mine = l < C::QW;
    const uint32_t ab0 = above[mine ? l : 0];
    const uint32_t as0 = pub ? above_s[mine ? l : 0] : 0u;
    const bool adv = mine && ab0 >= (uint32_t)k && tau_v < m - 1;
    const bool advs = mine && as0 >= (uint32_t)ks && taus_v < m - 1;
    if (__ballot(adv || advs) == 0) return;
    if (adv || advs) {
      const int lq = lane_here();
      if (adv) {
        uint32_t ab = ab0;
        int t = tau_v;
        while (ab >= (uint32_t)k && t < m - 1) {
          ++t;
          ab -= hist[lq * m + t];
        }
        move_tau(lq, t, ab);
      }
      if (advs) {
        uint32_t ab = as0;
        int t = taus_v;
        while (ab >= (uint32_t)ks && t < m - 1) {
          ++t;
          ab -= hist[lq * m + t];
        }
        above_s[lq] = ab;
        qs[lq].ups = up_of(t);
        taus_v = t;
        // (bins above 254 publish as 254: a lower bin is still a lower bound)
        __hip_atomic_store(pub + (int64_t)(qbase + lq) * 8 + split, (uint8_t)(min(t, 254) + 1), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    update_gates();
  }

  // Query of item it in lane half h, with a run-time item index.
  __device__ __forceinline__ static int item_query(int it, int h) {
    const int s = it % C::GPQ, g = it / C::GPQ, i = g % 4, mt = (g / 4) % C::MT;
    return (32 * mt + 8 * i + 4 * h + s * C::H) / C::H;
  }

  __device__ __forceinline__ void finish(uint32_t* cnt, uint32_t* hist_out) {
    if (qlen != 0) drain();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    const int l = lane_id();
    for (int q = 0; q < C::QW; ++q) {
      const int t = qbase + q;
      if (t >= nq) break;
      if (!row_on(t)) continue;
      const int64_t u = (int64_t)t * S + split;
      for (int b = l; b < m; b += kWave) hist_out[u * m + b] = hist[q * m + b];
    }
    if (l < C::QW && row_on(qbase + l)) cnt[(int64_t)(qbase + l) * S + split] = tail[l];
  }
};

// ---------------------------------------------------------------------------
// Kernels
// ---------------------------------------------------------------------------
template <class C, bool FAR>
__global__ __launch_bounds__(C::NTHREADS) void k_sample(ScoreArgs a, const int32_t* list, int ns, float* samp,
                                                        int slice) {
  extern __shared__ __align__(16) uint8_t lds[];
  const int q0 = blockIdx.x * C::QT, wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave),
            qbase = q0 + wave * C::QW;
  const int kb = blockIdx.y * slice, ke = min(kb + slice, ns);
  WaveQ<C> wq;
  load_q<C>(wq, a, qbase);
  DenseSink<C> sink{samp, ns, qbase, a.nq};
  wg_scan<C>(a, SrcListT<FAR>{list}, kb, ke, lds, wq, sink);
}

template <class C>
__global__ __launch_bounds__(C::NTHREADS) void k_dense(ScoreArgs a, float* out, int64_t ld, int slice) {
  extern __shared__ __align__(16) uint8_t lds[];
  const int q0 = blockIdx.x * C::QT, wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave),
            qbase = q0 + wave * C::QW;
  const int kb = blockIdx.y * slice, ke = min(kb + slice, a.nk);
  WaveQ<C> wq;
  load_q<C>(wq, a, qbase);
  DenseSink<C> sink{out, ld, qbase, a.nq};
  wg_scan<C>(a, SrcContig{}, kb, ke, lds, wq, sink);
}

// LDS of the fused scan besides the tile ring and the histograms: the
// per-query records of the grouped filter
template <class C>
constexpr int fused_sink_lds() {
  if constexpr (C::GROUPED) return C::WAVES * GroupedSink<C>::kLdsPerWave;
  else return 0;
}

template <class C>
__global__ __launch_bounds__(C::NTHREADS) void k_fused(ScoreArgs a, const RowParam* params, int S, int L, int cap,
                                                       int m, int k, uint8_t* pub, uint32_t* cnt,
                                                       uint32_t* hist_out, int2* cand, const int32_t* rflag,
                                                       const uint32_t* qctl) {
  extern __shared__ __align__(16) uint8_t lds[];
  uint32_t* hist = reinterpret_cast<uint32_t*>(lds + C::SCAN_LDS + fused_sink_lds<C>());
  // three words of block state after the histograms
  int* emax = reinterpret_cast<int*>(hist + C::QT * m);
  int* smin = emax + 1;
  int* anyon = emax + 2;
  const int tile = blockIdx.x / S, split = blockIdx.x - tile * S;
  const int q0 = tile * C::QT, wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave),
            qbase = q0 + wave * C::QW;
  // second filter pass: nothing queued
  if (rflag && qctl[1] == 0u) return;
  const bool on = threadIdx.x < C::QT && q0 + (int)threadIdx.x < a.nq && (!rflag || rflag[q0 + threadIdx.x]);
  for (int i = threadIdx.x; i < C::QT * m; i += C::NTHREADS) hist[i] = 0u;
  if (threadIdx.x == 0) {
    *emax = 0;
    *smin = a.nk;
    *anyon = 0;
  }
  __syncthreads();
  if (on) {
    *anyon = 1;
    const RowRange rr = row_range(a.offs, a.starts, q0 + threadIdx.x, a.nk);
    if (rr.e > rr.s) {
      atomicMax(emax, rr.e);
      atomicMin(smin, rr.s);
    }
  }
  __syncthreads();
  if (*anyon == 0) return;  // block-uniform: none of the block's rows is scanned (second pass)
  // the split's keys within the union of the block's rows' ranges
  const int kb = max(split * L, *smin);
  const int ke = min(min(split * L + L, a.nk), *emax);
  WaveQ<C> wq;
  load_q<C>(wq, a, qbase);
  std::conditional_t<C::GROUPED, GroupedSink<C>, FusedSink<C>> sink;
  sink.hist = hist + wave * C::QW * m;
  if constexpr (C::GROUPED) {
    sink.bind(lds + C::SCAN_LDS + wave * GroupedSink<C>::kLdsPerWave);
    sink.kq0 = kb;
    // splits share thresholds through one byte per (row, split): up to 8 splits
    sink.pub = S > 1 && S <= 8 ? pub : nullptr;
  }
  sink.cand = cand;
  sink.rflag = rflag;
  sink.qbase = qbase;
  sink.nq = a.nq;
  sink.S = S;
  sink.split = split;
  sink.cap = cap;
  sink.m = m;
  sink.k = k;
  sink.init(a, params, ke);
  wg_scan<C>(a, SrcContig{}, kb, ke, lds, wq, sink);
  sink.finish(cnt, hist_out);
}

// LDS bytes of the fallback's batch: the slot map of the tile's rows and the
// batch's rows.
template <class C>
constexpr int fallback_meta_lds() { return ((C::QT + 15) & ~15) + kMaxFallbackBatch * 4 + 16; }

// Exact fallback of the queued rows: dense re-score of each row's visible keys
// into scratch, then radix select, in split mode (few rows: each row's keys
// cut into chunks over many blocks, each selecting its chunk's top-k, the
// last one merging them), dense mode (the queued rows' tiles scored once in
// (tile, key slice) items; the selection is launch_fallback_rows') or
// whole-row mode (see launch_fused_fallback).
template <class C>
__global__ __launch_bounds__(C::NTHREADS) void k_fused_fallback(ScoreArgs a, int k, uint32_t flags, uint32_t* qctl,
                                                                const int32_t* queue, int32_t* fbflag, int batch,
                                                                int slots, size_t meta_off, float* scratch,
                                                                int32_t* cidx, float* cscore, int32_t* out_i,
                                                                float* out_s) {
  extern __shared__ __align__(16) uint8_t lds[];
  int8_t* smap = reinterpret_cast<int8_t*>(lds + meta_off);            // [QT]
  int* brow = reinterpret_cast<int*>(lds + meta_off + ((C::QT + 15) & ~15));  // [kMaxFallbackBatch]
  int* bn = brow + kMaxFallbackBatch;  // [0] rows of the pass, [1] select after the pass
  const uint32_t n = qctl[0];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  if (fbflag && fallback_dense(n, a.nq, gridDim.x, slots, a.nk, C::QT)) {
    // dense mode: items (tile x, slice y), consecutive items on the same
    // slice; queued row t of tile x goes to scratch row t (slot t - q0)
    const int tiles = (a.nq + C::QT - 1) / C::QT, nsl = (a.nk + kDenseSlice - 1) / kDenseSlice;
    for (int item = blockIdx.x; item < tiles * nsl; item += gridDim.x) {
      const int q0 = (item % tiles) * C::QT, y = item / tiles;
      if (threadIdx.x == 0) {
        brow[0] = INT_MAX;  // the union of the queued rows' visible ranges
        brow[1] = 0;
      }
      __syncthreads();
      if (threadIdx.x < C::QT) {
        const int t = q0 + (int)threadIdx.x;
        const bool on = t < a.nq && fbflag[t] == 1;
        smap[threadIdx.x] = on ? (int8_t)threadIdx.x : (int8_t)-1;
        if (on) {
          const RowRange rr = row_range(a.offs, a.starts, t, a.nk);
          if (rr.e > rr.s) {
            atomicMin(&brow[0], rr.s);
            atomicMax(&brow[1], rr.e);
          }
        }
      }
      __syncthreads();
      const int kb = max(y * kDenseSlice, brow[0]), ke = min(y * kDenseSlice + kDenseSlice, brow[1]);
      if (kb < ke) {  // block-uniform
        const int qbase = q0 + wave * C::QW;
        WaveQ<C> wq;
        load_q<C>(wq, a, qbase);
        RowSink<C> sink{scratch + (int64_t)q0 * a.nk, a.nk, smap, qbase, q0};
        wg_scan<C>(a, SrcContig{}, kb, ke, lds, wq, sink);
      }
      __syncthreads();  // smap and the range are rewritten by the next item
    }
    return;
  }
  const int chunks = fallback_chunks(n, gridDim.x, slots, a.nk);
  const bool split = chunks > 1;
  // split: block = (queue entry, chunk of that row's visible keys), one pass;
  // whole rows: the first slots / batch blocks, each with its own scratch
  // rows, take queue entries from a shared cursor (a block whose row another
  // block already took moves on at once)
  if ((int)blockIdx.x >= (split ? (int)n * chunks : slots / batch)) return;
  const int e = split ? (int)blockIdx.x / chunks : 0, c = split ? (int)blockIdx.x - e * chunks : 0;
  float* sblk = scratch + (int64_t)(split ? e : (int)blockIdx.x * batch) * a.nk;
  for (int pass = 0;; ++pass) {
    // the pass's rows: split, the entry's row; whole rows, the entry's row
    // unless another block took it with its own tile, then other queued rows
    // of the tile that no block has taken yet
    if (threadIdx.x == 0) {
      int nb = -1;  // nothing left
      if (split) {
        if (pass == 0) {
          brow[0] = queue[e];
          nb = 1;
        }
      } else {
        const uint32_t r = atomicAdd(&qctl[kQctlCursor], 1u);
        if (r < n) {
          nb = 0;
          const int row = queue[r];
          if (!fbflag || atomicExch(&fbflag[row], 2) == 1) {
            brow[nb++] = row;
            if (fbflag) {
              const int q0 = (row / C::QT) * C::QT, qe = min(q0 + C::QT, a.nq);
              for (int t = q0; t < qe && nb < batch; ++t)
                if (t != row && atomicCAS(&fbflag[t], 1, 2) == 1) brow[nb++] = t;
            }
          }
        }
      }
      bn[0] = nb;
    }
    for (int i = threadIdx.x; i < C::QT; i += C::NTHREADS) smap[i] = -1;
    __syncthreads();
    const int nb = bn[0];
    if (nb < 0) return;  // block-uniform
    if (nb == 0) {
      __syncthreads();  // every thread has read bn[0] before the next entry rewrites it
      continue;
    }
    const int q0 = (brow[0] / C::QT) * C::QT, qbase = q0 + wave * C::QW;
    if (threadIdx.x < nb) smap[brow[threadIdx.x] - q0] = (int8_t)threadIdx.x;
    // keys of the pass: split, the chunk; whole rows, the union of the rows'
    // ranges (each row selects from its own)
    int kb = a.nk, ke = 0, rs = 0, len = 0, per = 0;
    if (split) {
      const RowRange rr = row_range(a.offs, a.starts, brow[0], a.nk);
      rs = rr.s;
      len = rr.e > rr.s ? rr.e - rr.s : 0;
      per = ((len + chunks - 1) / chunks + C::KT - 1) / C::KT * C::KT;
      kb = min(rs + c * per, rs + len);
      ke = min(kb + per, rs + len);
    } else {
      for (int j = 0; j < nb; ++j) {
        const RowRange rr = row_range(a.offs, a.starts, brow[j], a.nk);
        if (rr.e > rr.s) {
          kb = min(kb, rr.s);
          ke = max(ke, rr.e);
        }
      }
    }
    __syncthreads();
    WaveQ<C> wq;
    load_q<C>(wq, a, qbase);
    RowSink<C> sink{sblk, a.nk, smap, qbase, q0};
    wg_scan<C>(a, SrcContig{}, kb, ke, lds, wq, sink);
    __threadfence_block();
    __syncthreads();
    if (split) {
      // the chunk's top-k to the row's candidates; the last chunk selects
      const int t = brow[0];
      const int64_t cb = (int64_t)e * chunks * k;
      split_fallback_select<C::NTHREADS>(sblk, rs, len, per, chunks, c, kb, ke, k, cidx + cb, cscore + cb,
                                         &qctl[kQctlDone + e], out_i + (int64_t)t * k, out_s + (int64_t)t * k,
                                         flags & LT_SORTED_OUTPUT, lds, &bn[1]);
    } else {
      for (int j = 0; j < nb; ++j) {
        const int t = brow[j];
        const RowRange rr = row_range(a.offs, a.starts, t, a.nk);
        radix_select_row<C::NTHREADS>(sblk + (int64_t)j * a.nk + rr.s, rr.e - rr.s, k, out_i + (int64_t)t * k,
                                      out_s + (int64_t)t * k, flags & LT_SORTED_OUTPUT, lds, rr.s);
        __syncthreads();
      }
    }
    __syncthreads();  // brow and bn are rewritten by the next pass
  }
}

// ---------------------------------------------------------------------------
// Compiled variants and dispatch
// ---------------------------------------------------------------------------
//            dtype   H   d  QW NT WAVES RELU
#define LT_VARIANTS(X)                   \
  X(DT_F32, 4, 64, 8, 2, 4, true)        \
  X(DT_F32, 1, 64, 32, 2, 4, true)       \
  X(DT_F32, 1, 64, 32, 2, 4, false)      \
  X(DT_BF16, 64, 128, 1, 2, 8, true)     \
  X(DT_BF16, 4, 128, 8, 2, 4, true)      \
  X(DT_BF16, 1, 128, 32, 2, 8, true)     \
  X(DT_BF16, 1, 128, 32, 2, 8, false)    \
  X(DT_FP8, 64, 128, 1, 2, 8, true)

// unitw: the inner-product one-head shapes without head weights take the
// UNITW variant (same results, no epilogue arithmetic)
template <class F>
static bool with_cfg(int dt, int mode, int h, int d, bool unitw, F&& f) {
  const bool relu = mode == LT_SCORE_DSA;
#define LT_CASE(DT, H, D, QW, NT, WV, RELU)                                  \
  if (dt == DT && h == H && d == D && relu == RELU) {                        \
    if constexpr (H == 1 && !RELU) {                                         \
      if (unitw) {                                                           \
        f.template operator()<Cfg<DT, H, D, QW, NT, WV, RELU, true>>();      \
        return true;                                                         \
      }                                                                      \
    }                                                                        \
    f.template operator()<Cfg<DT, H, D, QW, NT, WV, RELU>>();                \
    return true;                                                             \
  }
  LT_VARIANTS(LT_CASE)
#undef LT_CASE
  return false;
}

ScoreShape score_shape(int dtype, int mode, int h, int d) {
  ScoreShape s{0, 0, 0, 0, 0, 0, 0};
  const bool found = with_cfg(dtype, mode, h, d, false, [&]<class C>() {
    s.supported = 1;
    s.arrival_order = C::GROUPED ? 1 : 0;
    s.queries_per_block = C::QT;
    s.keys_per_step = C::KT;
    s.threads = C::NTHREADS;
    s.scan_lds = C::SCAN_LDS + fused_sink_lds<C>();
  });
  return found ? s : wide_shape(dtype, mode, h, d);
}

static constexpr int kSlice = 8192;   // positions per block in the sample / dense scorers
static constexpr int kSampleBlocks = 256;  // the sample scorer aims at one block per CU at least

hipError_t launch_sample_scores(const ScoreArgs& a, const int32_t* list, int ns, float* samp, hipStream_t st) {
  if (wide_shape(a.dtype, a.mode, a.h, a.d).supported) return launch_wide_sample(a, list, ns, samp, st);
  hipError_t err = hipErrorInvalidValue;
  with_cfg(a.dtype, a.mode, a.h, a.d, a.w == nullptr, [&]<class C>() {
    // few query tiles (a short chunk): cut the sample into more slices so
    // that the launch still covers the GPU
    const int tiles = (a.nq + C::QT - 1) / C::QT;
    const int want = tiles > 0 ? (kSampleBlocks + tiles - 1) / tiles : 1;
    int slice = (ns + want - 1) / want;
    slice = ((slice + C::KT - 1) / C::KT) * C::KT;
    slice = slice < C::KT ? C::KT : (slice > kSlice ? kSlice : slice);
    dim3 grid(tiles, (ns + slice - 1) / slice);
    if (grid.x == 0 || grid.y == 0) {
      err = hipSuccess;
      return;
    }
    // a buffer descriptor reaches 4 GiB of keys; larger key arrays gather
    // through per-lane global addresses
    if ((uint64_t)a.nk * C::ROWB < (1ull << 32))
      hipLaunchKernelGGL((k_sample<C, false>), grid, dim3(C::NTHREADS), C::SCAN_LDS, st, a, list, ns, samp, slice);
    else
      hipLaunchKernelGGL((k_sample<C, true>), grid, dim3(C::NTHREADS), C::SCAN_LDS, st, a, list, ns, samp, slice);
    err = hipGetLastError();
  });
  return err;
}

hipError_t launch_dense_scores(const ScoreArgs& a, float* out, int64_t ld, hipStream_t st) {
  if (wide_shape(a.dtype, a.mode, a.h, a.d).supported) return launch_wide_dense(a, out, ld, st);
  hipError_t err = hipErrorInvalidValue;
  with_cfg(a.dtype, a.mode, a.h, a.d, a.w == nullptr, [&]<class C>() {
    dim3 grid((a.nq + C::QT - 1) / C::QT, (a.nk + kSlice - 1) / kSlice);
    if (grid.x == 0 || grid.y == 0) {
      err = hipSuccess;
      return;
    }
    hipLaunchKernelGGL(k_dense<C>, grid, dim3(C::NTHREADS), C::SCAN_LDS, st, a, out, ld, kSlice);
    err = hipGetLastError();
  });
  return err;
}

// Published bins of the rows' splits start at the sample's (stored + 1).
__global__ void k_pub_init(const RowParam* params, int nq, uint64_t* pub) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nq; i += (int64_t)gridDim.x * blockDim.x)
    pub[i] = 0x0101010101010101ull * (uint64_t)(uint8_t)(min(params[i].tau0, 254) + 1);
}

hipError_t launch_fused_scan(const ScoreArgs& a, const RowParam* params, int S, int L, int cap, int m, int k,
                             int* pub, uint32_t* cnt, uint32_t* hist, int2* cand, const int32_t* rflag,
                             const uint32_t* qctl, hipStream_t st) {
  hipError_t err = hipErrorInvalidValue;
  with_cfg(a.dtype, a.mode, a.h, a.d, a.w == nullptr, [&]<class C>() {
    const int tiles = (a.nq + C::QT - 1) / C::QT;
    if (tiles == 0) {
      err = hipSuccess;
      return;
    }
    if (C::GROUPED && S > 1 && S <= 8) {
      hipLaunchKernelGGL(k_pub_init, dim3((a.nq + 255) / 256), dim3(256), 0, st, params, a.nq,
                         reinterpret_cast<uint64_t*>(pub));
      if ((err = hipGetLastError()) != hipSuccess) return;
    }
    const size_t lds = C::SCAN_LDS + fused_sink_lds<C>() + (size_t)C::QT * m * 4 + 16;
    if (lds > 65536)
      (void)hipFuncSetAttribute((const void*)k_fused<C>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(k_fused<C>, dim3(tiles * S), dim3(C::NTHREADS), lds, st, a, params, S, L, cap, m, k,
                       reinterpret_cast<uint8_t*>(pub), cnt, hist, cand, rflag, qctl);
    err = hipGetLastError();
  });
  return err;
}

hipError_t launch_fused_fallback(const ScoreArgs& a, int k, uint32_t flags, uint32_t* qctl, const int32_t* queue,
                                 int32_t* fbflag, int batch, int slots, float* scratch, int32_t* cidx, float* cscore,
                                 int32_t* out_i, float* out_s, hipStream_t st) {
  if (wide_shape(a.dtype, a.mode, a.h, a.d).supported)
    return launch_wide_fallback(a, k, flags, qctl, queue, slots, scratch, cidx, cscore, out_i, out_s, st);
  hipError_t err = hipErrorInvalidValue;
  with_cfg(a.dtype, a.mode, a.h, a.d, a.w == nullptr, [&]<class C>() {
    size_t lds = C::SCAN_LDS;
    const size_t rl = radix_lds_bytes(k);
    if (rl > lds) lds = rl;
    const size_t meta = (lds + 15) & ~(size_t)15;
    lds = meta + fallback_meta_lds<C>();
    if (lds > 65536)
      (void)hipFuncSetAttribute((const void*)k_fused_fallback<C>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    const int b = batch < 1 ? 1 : (batch > kMaxFallbackBatch ? kMaxFallbackBatch : batch);
    hipLaunchKernelGGL(k_fused_fallback<C>, dim3(kFallbackGrid), dim3(C::NTHREADS), lds, st, a, k, flags, qctl,
                       queue, fbflag, b, slots, meta, scratch, cidx, cscore, out_i, out_s);
    err = hipGetLastError();
  });
  return err;
}

}  // namespace lt
