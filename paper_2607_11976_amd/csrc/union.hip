// LiteDSA's group union and per-query membership masks (sec. 3.3). One
// block per group of consecutive queries:
//  1. the group's keys (every list, padding dropped) go into LDS and are
//     sorted ascending (bitonic sort of the descending order of ~key, which
//     sends the dropped entries, mapped to 0, last);
//  2. the first of each run of equal keys takes the next union slot (ordered
//     compaction with a block scan), so the union is ascending and distinct;
//  3. for each query, every key of its list finds its union slot by binary
//     search and sets that bit of the query's mask, built in LDS with atomic
//     ORs and then written out.
// The paper dedups through a bitmap over the whole key space; sorting the
// group's at most LT_UNION_MAX entries needs LDS bounded by the group, not by
// the context length, and yields the same ascending union.
#include <algorithm>

#include "internal.hpp"
#include "select_dev.hpp"

namespace lt {

constexpr int kUnionThreads = 1024;

__global__ __launch_bounds__(kUnionThreads) void k_dsa_union(const int32_t* idx, int64_t ld, int nq, int k, int group,
                                                              int32_t* uidx, int32_t* ucount, uint32_t* mask) {
  extern __shared__ __align__(16) uint32_t lds_u[];
  __shared__ uint32_t tmp[kUnionThreads / kWave];
  const int g = blockIdx.x, t0 = g * group, nt = min(group, nq - t0);
  const int n = group * k, P = next_pow2(n), W = (n + 31) / 32;
  uint32_t* a = lds_u;          // [P] sort buffer, then the union
  uint32_t* mw = lds_u + P;     // [W] mask of one query
  const int tid = threadIdx.x;

  // 1. load (rows past the last query and negative entries are dropped)
  for (int i = tid; i < P; i += kUnionThreads) {
    int v = -1;
    if (i < n) {
      const int r = i / k, j = i - r * k;
      if (r < nt) v = idx[(int64_t)(t0 + r) * ld + j];
    }
    a[i] = v >= 0 ? ~(uint32_t)v : 0u;
  }
  __syncthreads();
  bitonic_sort_desc<kUnionThreads>(a, P);

  // 2. ordered compaction of the first entry of every run; a[] is rewritten
  //    in place: a round writes slots <= its positions, after all its reads,
  //    and the one earlier position a round reads (i0 - 1, which the round
  //    before may have overwritten) is carried in `carry`
  __shared__ uint32_t carry;
  uint32_t base = 0;
  for (int i0 = 0; i0 < P; i0 += kUnionThreads) {
    const int i = i0 + tid;
    const uint32_t x = i < P ? a[i] : 0u;
    const uint32_t prev = (i == 0 || i >= P) ? 0u : (tid == 0 ? carry : a[i - 1]);
    const bool first = x != 0u && x != prev;
    uint32_t total;
    const uint32_t ex = block_scan_excl<kUnionThreads>(first ? 1u : 0u, tmp, &total);
    __syncthreads();  // every read of this round precedes any write
    if (tid == kUnionThreads - 1) carry = x;
    if (first) a[base + ex] = ~x;  // the key itself
    base += total;
    __syncthreads();
  }
  const int count = (int)base;
  int32_t* urow = uidx + (int64_t)g * n;
  for (int i = tid; i < n; i += kUnionThreads) urow[i] = i < count ? (int32_t)a[i] : -1;
  if (tid == 0) ucount[g] = count;

  // 3. membership masks, one query at a time
  for (int r = 0; r < nt; ++r) {
    for (int w = tid; w < W; w += kUnionThreads) mw[w] = 0u;
    __syncthreads();
    for (int j = tid; j < k; j += kUnionThreads) {
      const int v = idx[(int64_t)(t0 + r) * ld + j];
      if (v < 0) continue;
      // lower bound of v in the ascending union a[0, count); v is present
      int lo = 0, hi = count;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if ((int)a[mid] < v) lo = mid + 1;
        else hi = mid;
      }
      atomicOr(&mw[lo >> 5], 1u << (lo & 31));
    }
    __syncthreads();
    uint32_t* mrow = mask + (int64_t)(t0 + r) * W;
    for (int w = tid; w < W; w += kUnionThreads) mrow[w] = mw[w];
    __syncthreads();
  }
}

size_t union_lds_bytes(int group, int k) {
  const int n = group * k;
  return ((size_t)next_pow2(n) + (size_t)(n + 31) / 32) * 4;
}

hipError_t launch_dsa_union(const int32_t* idx, int64_t ld, int nq, int k, int group, int32_t* uidx, int32_t* ucount,
                            uint32_t* mask, hipStream_t st) {
  const int groups = (nq + group - 1) / group;
  if (groups == 0) return hipSuccess;
  const size_t lds = union_lds_bytes(group, k);
  if (lds > 65536)
    (void)hipFuncSetAttribute((const void*)k_dsa_union, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  hipLaunchKernelGGL(k_dsa_union, dim3(groups), dim3(kUnionThreads), lds, st, idx, ld, nq, k, group, uidx, ucount,
                     mask);
  return hipGetLastError();
}

}  // namespace lt
