// Tiles of a delta chain, for the one-pass chain apply (apply.hip).
//
// A chain D_1..D_K (oldest first, each strictly increasing) is cut into
// value ranges: tile t holds the indices from boundary b_t up to b_{t+1}
// (tile 0 from minus infinity, the last to plus infinity), so every entry
// of every delta lies in exactly one tile.  A split kernel finds where
// each tile starts in each delta.  A workgroup then stages its tile's runs
// in LDS and gives every entry its position in the merged order of all
// runs (ties: older delta first), so that of equal indices the newest
// comes last.
#pragma once

#include "delta_internal.h"

namespace aurora {

// The deltas' addresses come from a table in memory, so the compiler
// cannot tell they are global; flat accesses would also count against the
// LDS wait counter, so the chain kernels use these global-space views.
template <typename T>
__device__ __forceinline__ const __attribute__((address_space(1))) T* gview(const T* p) {
  return (const __attribute__((address_space(1))) T*)p;
}

constexpr int kChainThreads = 256;
constexpr int kChainLoads = 8;   // staging loads per thread in flight
static_assert(kChainLds <= 4096 && kChainMaxDeltas <= 16,
              "a merged position holds (delta << 12) | staged entry in 16 bits");

struct ChainSmem {
  int64_t idx[kChainLds];                  // the tile's runs, one after another
  uint16_t perm[kChainLds];                // merged position -> (delta << 12) | entry
  ChainDelta d[kChainMaxDeltas];
  uint64_t start[kChainMaxDeltas];         // each run's first entry in its delta
  uint32_t off[kChainMaxDeltas + 1];       // run offsets in the tile's order
};

// Block-wide (barriers): the tile's run bounds into LDS; returns the
// tile's entries, capped at 2^32 - 1 (more, or unsorted input, sets bad).
__device__ __forceinline__ uint32_t chain_tile_setup(const ChainRuns& r, uint64_t t,
                                                     ChainSmem& s, bool& bad) {
  const uint32_t K = r.K;
  if (threadIdx.x < K) {
    const uint32_t k = threadIdx.x;
    const uint64_t p0 = r.pos[t * K + k];
    uint64_t p1 = r.pos[(t + 1) * K + k];
    if (p1 < p0) {   // only unsorted input gets here
      bad = true;
      p1 = p0;
    }
    if (p1 - p0 >= 0xFFFFFFFFull) bad = true;
    s.d[k] = r.deltas[k];
    s.start[k] = p0;
    s.off[k + 1] = (uint32_t)(p1 - p0 < 0xFFFFFFFFull ? p1 - p0 : 0xFFFFFFFFull);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t acc = 0;
    s.off[0] = 0;
    for (uint32_t k = 0; k < K; ++k) {
      acc += s.off[k + 1];
      if (acc >= 0xFFFFFFFFull) bad = true;
      s.off[k + 1] = (uint32_t)(acc < 0xFFFFFFFFull ? acc : 0xFFFFFFFFull);
    }
  }
  __syncthreads();
  return s.off[K];
}

// Entries of the sorted run x[0, n) below v (upper: at most v).
template <typename Ptr>
__device__ __forceinline__ uint32_t run_rank(Ptr x, uint32_t n, int64_t v, bool upper) {
  uint32_t lo = 0, hi = n;
  while (lo < hi) {
    const uint32_t mid = (lo + hi) >> 1;
    if (x[mid] < v || (upper && x[mid] == v)) lo = mid + 1; else hi = mid;
  }
  return lo;
}

// Block-wide, total <= kChainLds: stages the runs' indices (kChainLoads
// loads per thread in flight), then writes the merged order into s.perm:
// an entry's position is its place in its own run plus, in every other
// run, the entries below it (newer runs) or at most it (older runs).
// Sorted runs give a permutation; unsorted ones set bad (positions stay
// inside the array).
__device__ __forceinline__ void chain_stage_rank(uint32_t K, uint32_t total, ChainSmem& s,
                                                 bool& bad) {
  {
    uint32_t k = 0;
    for (uint32_t q0 = threadIdx.x; q0 < total; q0 += kChainThreads * kChainLoads) {
      int64_t x[kChainLoads];
#pragma unroll
      for (int u = 0; u < kChainLoads; ++u) {
        const uint32_t q = q0 + kChainThreads * u;
        x[u] = 0;
        if (q < total) {
          while (q >= s.off[k + 1]) ++k;
          x[u] = gview(s.d[k].idx)[s.start[k] + (q - s.off[k])];
        }
      }
#pragma unroll
      for (int u = 0; u < kChainLoads; ++u) {
        const uint32_t q = q0 + kChainThreads * u;
        if (q < total) s.idx[q] = x[u];
      }
    }
  }
  __syncthreads();
  uint32_t k = 0;
  for (uint32_t q = threadIdx.x; q < total; q += kChainThreads) {
    while (q >= s.off[k + 1]) ++k;
    const int64_t x = s.idx[q];
    if (q + 1 < s.off[k + 1] && s.idx[q + 1] <= x) bad = true;   // unsorted run
    uint32_t pos = q - s.off[k];
    for (uint32_t k2 = 0; k2 < K; ++k2)
      if (k2 != k) pos += run_rank(s.idx + s.off[k2], s.off[k2 + 1] - s.off[k2], x, k2 < k);
    s.perm[pos < total ? pos : total - 1] = (uint16_t)((k << 12) | q);
  }
  __syncthreads();
}

// The entry at merged position p (p < total): its delta k and staged slot
// q, checked (only unsorted input can give a bad one); kept when the next
// position holds another index.
__device__ __forceinline__ bool chain_entry(const ChainSmem& s, uint32_t K, uint32_t total,
                                            uint32_t p, uint32_t& k, uint32_t& q, bool& keep) {
  const uint32_t code = s.perm[p];
  k = code >> 12;
  q = code & 0xFFFu;
  if (k >= K || q < s.off[k] || q >= s.off[k + 1]) return false;
  keep = p + 1 == total || s.idx[s.perm[p + 1] & 0xFFFu] != s.idx[q];
  return true;
}

}  // namespace aurora
