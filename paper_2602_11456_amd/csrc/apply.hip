// Delta application on gfx950: write each kept word back into the flat
// storage of the rollout copy, w[idx[k]] = val[k] (AuroraRL Sec. 5.1 and
// Sec. 5.2: an in-place flat scatter at an end-of-batch safe point).
//
// The value stream holds the new words themselves, so the scatter assigns
// rather than adds: the result is bit-exact and applying a delta twice
// changes nothing.  Indices are distinct, so no two lanes write one word
// and no atomics are needed.
#include "chain.h"
#include "delta_internal.h"

namespace aurora {

constexpr int kApplyThreads = 256;
constexpr int kApplyWaves = kApplyThreads / 64;
constexpr int kApplyPerLane = 8;
constexpr int kApplyPerWave = 64 * kApplyPerLane;
// Scattered stores marked non-temporal (streamed past the caches).
constexpr bool kNtScatter = true;

__device__ __forceinline__ void flag_error(uint32_t* err) {
  if (err) __hip_atomic_fetch_or(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The tensor addresses of the multi-tensor kernels come from a table in
// memory, so the store goes through a global-space view (a flat store would
// also count against the LDS wait counter).
__device__ __forceinline__ void store_word(uint16_t* p, uint16_t v) {
  __attribute__((address_space(1))) uint16_t* g = (__attribute__((address_space(1))) uint16_t*)p;
  if (kNtScatter)
    __builtin_nontemporal_store(v, g);
  else
    *g = v;
}

// Wavefront w of the grid covers entries [512 w, 512 (w + 1)) (grid-stride):
// lane l handles entries 512 w + 64 u + l, u = 0..7, so every load reads 64
// consecutive entries and every store instruction writes 64 consecutive
// (sorted) entries, i.e. a short stretch of the weights.
template <typename IdxT>
__global__ __launch_bounds__(kApplyThreads) void apply_kernel(uint16_t* __restrict__ w, uint64_t n,
                                                              const IdxT* __restrict__ idx,
                                                              const uint16_t* __restrict__ val,
                                                              uint64_t count, uint32_t* err) {
  const uint32_t lane = threadIdx.x & 63;
  const uint64_t waves = (uint64_t)gridDim.x * kApplyWaves;
  bool bad = false;
  for (uint64_t wv = (uint64_t)blockIdx.x * kApplyWaves + (threadIdx.x >> 6);
       wv * kApplyPerWave < count; wv += waves) {
    const uint64_t k0 = wv * kApplyPerWave + lane;
    int64_t i[kApplyPerLane];
    uint16_t v[kApplyPerLane];
#pragma unroll
    for (int u = 0; u < kApplyPerLane; ++u) {
      const uint64_t k = k0 + 64 * u;
      i[u] = k < count ? (int64_t)idx[k] : -1;
      v[u] = k < count ? val[k] : 0;
    }
#pragma unroll
    for (int u = 0; u < kApplyPerLane; ++u) {
      if (k0 + 64 * u >= count) continue;
      if (i[u] >= 0 && (uint64_t)i[u] < n)
        store_word(w + i[u], v[u]);
      else
        bad = true;
    }
  }
  if (bad) flag_error(err);
}

// Global index -> (tensor, local index) over T tensors with bases[0..T]
// (bases[t] = first global index of tensor t, bases[T] = total).
__device__ __forceinline__ uint32_t find_tensor(const uint64_t* bases, uint32_t T, uint64_t g) {
  uint32_t lo = 0, hi = T;   // answer in [lo, hi): bases[lo] <= g < bases[hi]
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) >> 1;
    if (bases[mid] <= g) lo = mid; else hi = mid;
  }
  return lo;
}

__global__ __launch_bounds__(kApplyThreads) void apply_multi_kernel(
    const uint64_t* __restrict__ bases, uint16_t* const* __restrict__ ptrs, uint32_t T,
    const int64_t* __restrict__ idx, const uint16_t* __restrict__ val, uint64_t count,
    uint32_t* err) {
  const uint32_t lane = threadIdx.x & 63;
  const uint64_t waves = (uint64_t)gridDim.x * kApplyWaves;
  const uint64_t total = bases[T];
  bool bad = false;
  uint32_t t = 0;
  uint64_t lo = 1, hi = 0;   // empty range: forces a search first
  uint16_t* base_ptr = nullptr;
  for (uint64_t wv = (uint64_t)blockIdx.x * kApplyWaves + (threadIdx.x >> 6);
       wv * kApplyPerWave < count; wv += waves) {
    const uint64_t k0 = wv * kApplyPerWave + lane;
    int64_t i[kApplyPerLane];
    uint16_t v[kApplyPerLane];
#pragma unroll
    for (int u = 0; u < kApplyPerLane; ++u) {
      const uint64_t k = k0 + 64 * u;
      i[u] = k < count ? idx[k] : -1;
      v[u] = k < count ? val[k] : 0;
    }
#pragma unroll
    for (int u = 0; u < kApplyPerLane; ++u) {
      if (k0 + 64 * u >= count) continue;
      const int64_t g = i[u];
      if (g < 0 || (uint64_t)g >= total) {
        bad = true;
        continue;
      }
      if (!((uint64_t)g >= lo && (uint64_t)g < hi)) {
        t = find_tensor(bases, T, (uint64_t)g);
        lo = bases[t];
        hi = bases[t + 1];
        base_ptr = ptrs[t];
      }
      store_word(base_ptr + ((uint64_t)g - lo), v[u]);
    }
  }
  if (bad) flag_error(err);
}

// ------------------------------------------------ catch-up in one pass
//
// Applies D_1..D_K (oldest first) so that every index gets the word of the
// newest delta holding it: the result of replaying the chain (Sec. 5.4) or
// of applying its composition, without forming the composed delta.  The
// tiles (chain.h) are cut at every S-th index of the largest delta, so a
// tile holds S of its entries and, for deltas of similar density, about
// as many of every other.  A tile whose runs fit in LDS is ranked into
// merged order and its kept words (the newest of equal indices) are stored
// in index order, as a composed delta would store them; a larger tile
// (deltas of very uneven density) searches newer runs in global memory and
// stores in run order.

__global__ void chain_split_kernel(ChainRuns r) {
  const uint64_t q = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= (r.tiles + 1) * r.K) return;
  const uint64_t b = q / r.K;
  const uint32_t k = (uint32_t)(q % r.K);
  const ChainDelta d = r.deltas[k];
  uint64_t p;
  if (b == 0) {
    p = 0;
  } else if (b == r.tiles) {
    p = d.n;
  } else {
    const int64_t v = gview(r.bsrc)[b * r.bstride];
    uint64_t lo = 0, hi = d.n;
    const auto x = gview(d.idx);
    while (lo < hi) {
      const uint64_t mid = (lo + hi) >> 1;
      if (x[mid] < v) lo = mid + 1; else hi = mid;
    }
    p = lo;
  }
  r.pos[q] = p;
}

hipError_t launch_chain_split(const ChainRuns& r, hipStream_t stream) {
  const uint64_t bounds = (r.tiles + 1) * r.K;
  hipLaunchKernelGGL(chain_split_kernel, dim3((uint32_t)((bounds + 255) / 256)), dim3(256), 0,
                     stream, r);
  return hipGetLastError();
}

constexpr int kChainPer = 8;   // entries per thread loaded before any is processed

// Stores word v at global index g of the tensor list (the lane caches the
// tensor it wrote last); false if g is outside the list.
struct TensorCursor {
  uint32_t t = 0;
  uint64_t lo = 1, hi = 0;   // empty range: forces a search first
  uint16_t* base = nullptr;
};
__device__ __forceinline__ bool store_global(const ChainArgs& a, uint64_t words, TensorCursor& c,
                                             int64_t g, uint16_t v) {
  if (g < 0 || (uint64_t)g >= words) return false;
  if (!((uint64_t)g >= c.lo && (uint64_t)g < c.hi)) {
    c.t = find_tensor(a.bases, a.T, (uint64_t)g);
    c.lo = a.bases[c.t];
    c.hi = a.bases[c.t + 1];
    c.base = a.ptrs[c.t];
  }
  store_word(c.base + ((uint64_t)g - c.lo), v);
  return true;
}

static_assert(kApplyThreads == kChainThreads, "the chain helpers assume 256 threads");

__global__ __launch_bounds__(kApplyThreads) void chain_apply_kernel(ChainArgs a) {
  __shared__ ChainSmem s;
  const uint32_t K = a.r.K;
  bool bad = false;
  const uint32_t total = chain_tile_setup(a.r, blockIdx.x, s, bad);
  const uint64_t words = a.bases[a.T];
  TensorCursor cur;
  if (total <= kChainLds) {   // uniform
    chain_stage_rank(K, total, s, bad);
    for (uint32_t p0 = threadIdx.x; p0 < total; p0 += kApplyThreads * kChainPer) {
      int64_t x[kChainPer];
      uint16_t v[kChainPer];
      bool keep[kChainPer];
#pragma unroll
      for (int u = 0; u < kChainPer; ++u) {
        const uint32_t p = p0 + kApplyThreads * u;
        keep[u] = false;
        x[u] = 0;
        v[u] = 0;
        uint32_t k, q;
        if (p < total) {
          if (!chain_entry(s, K, total, p, k, q, keep[u])) {
            bad = true;
            continue;
          }
          x[u] = s.idx[q];
          if (keep[u]) v[u] = gview(s.d[k].val)[s.start[k] + (q - s.off[k])];
        }
      }
#pragma unroll
      for (int u = 0; u < kChainPer; ++u)
        if (keep[u] && !store_global(a, words, cur, x[u], v[u])) bad = true;
    }
  } else {
    // A tile too large for LDS: each entry in turn, written unless a newer
    // run holds its index (binary search in global memory).
    uint32_t k = 0;
    for (uint32_t q = threadIdx.x; q < total; q += kApplyThreads) {
      while (q >= s.off[k + 1]) ++k;
      const uint64_t e = s.start[k] + (q - s.off[k]);
      const auto xs = gview(s.d[k].idx);
      const int64_t x = xs[e];
      if (q + 1 < s.off[k + 1] && xs[e + 1] <= x) bad = true;
      bool newer = false;
      for (uint32_t k2 = k + 1; k2 < K && !newer; ++k2) {
        const uint32_t n2 = s.off[k2 + 1] - s.off[k2];
        const auto r = gview(s.d[k2].idx) + s.start[k2];
        const uint32_t at = run_rank(r, n2, x, false);
        newer = at < n2 && r[at] == x;
      }
      if (!newer && !store_global(a, words, cur, x, gview(s.d[k].val)[e])) bad = true;
    }
  }
  if (bad) flag_error(a.err);
}

hipError_t launch_apply_chain(const ChainArgs& a, hipStream_t stream) {
  if (a.r.tiles == 0) return hipSuccess;
  hipError_t e = launch_chain_split(a.r, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(chain_apply_kernel, dim3((uint32_t)a.r.tiles), dim3(kApplyThreads), 0,
                     stream, a);
  return hipGetLastError();
}


// ------------------------------------------- dense deltas: tiles merged
//
// For a delta in increasing index order that touches most 64-byte lines of
// the weights (from about 1 word in 32), scattered 2-byte stores cost one
// partial-line write each, which the memory serves as a read-modify-write.
// Here every workgroup takes one tile of kMergeTile words of one tensor:
// it reads the tile (16-byte loads), finds the tile's slice of the delta
// (two 64-wide searches over the sorted indices, issued beside the tile's
// loads), patches the slice into the tile in LDS and writes the tile back
// whole.  Each word of the weights is read and written once, in full lines.

constexpr int kMergeTile = 16384;                      // words per tile
constexpr int kMergeVec = kMergeTile / 8 / kApplyThreads;   // 16-byte vectors per thread
constexpr int kMergeLoads = 4;                         // slice entries per thread in flight

typedef uint32_t mg_u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) mg_u32x4 mg_gv4;

// First position p in [lo, hi) of the sorted x with x[p] >= target (hi if
// none), by one wavefront: each round probes 64 evenly spaced positions.
__device__ __forceinline__ uint64_t wave_lower_bound(const int64_t* x, uint64_t lo, uint64_t hi,
                                                     int64_t target) {
  const uint32_t lane = threadIdx.x & 63;
  const auto g = gview(x);
  while (hi - lo > 64) {
    const uint64_t span = hi - lo;
    const uint64_t p = lo + span / 65 * (lane + 1) + span % 65 * (lane + 1) / 65;
    const uint32_t c = (uint32_t)__builtin_popcountll(__ballot(g[p] < target));
    const uint64_t nlo = c ? (uint64_t)__shfl((long long)p, (int)c - 1) + 1 : lo;
    const uint64_t nhi = c < 64 ? (uint64_t)__shfl((long long)p, (int)(c < 64 ? c : 63)) : hi;
    lo = nlo;
    hi = nhi;
  }
  const uint64_t p = lo + lane;
  const bool less = p < hi && g[p] < target;
  return lo + (uint64_t)__builtin_popcountll(__ballot(less));
}

// tile_first[t]: first tile of tensor t (tile_first[T] = all tiles).
struct MergeArgs {
  const uint64_t* bases;
  uint16_t* const* ptrs;
  const uint64_t* tile_first;
  uint32_t T;
  uint64_t tiles;
  const int64_t* idx;
  const uint16_t* val;
  uint64_t count;
  uint32_t* err;
};

__global__ __launch_bounds__(kApplyThreads) void apply_merge_kernel(MergeArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t s_w[kMergeTile];
  __shared__ uint64_t s_r[2];
  __shared__ uint32_t s_t;
  const uint64_t b = blockIdx.x;
  const uint32_t wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (wave == 0) {
    // the tensor of tile b: the last t with tile_first[t] <= b (tiles of
    // an empty tensor start where the next tensor's do, so no later t
    // qualifies).  Lane l probes lo + floor(n l / 64): lane 0 probes lo,
    // which always qualifies, and with n <= 64 every candidate is probed.
    uint32_t lo = 0, hi = a.T;   // tile_first[lo] <= b; the answer is in [lo, hi)
    while (hi - lo > 1) {
      const uint32_t n = hi - lo;
      const uint32_t p = lo + (uint32_t)(((uint64_t)n * lane) >> 6);
      const uint64_t m = __ballot(a.tile_first[p] <= b);   // a prefix of the lanes
      const uint32_t c = 63 - (uint32_t)__builtin_clzll(m);
      const uint32_t last = (uint32_t)__shfl((int)p, (int)c);
      const uint32_t next = (uint32_t)__shfl((int)p, (int)(c < 63 ? c + 1 : 63));
      lo = last;
      if (c < 63) hi = next;
    }
    if (lane == 0) s_t = lo;
  }
  __syncthreads();
  const uint32_t t = s_t;
  const uint64_t lo_w = (b - a.tile_first[t]) * kMergeTile;
  const uint64_t n_t = a.bases[t + 1] - a.bases[t];
  const uint64_t len = n_t - lo_w < (uint64_t)kMergeTile ? n_t - lo_w : kMergeTile;
  const uint64_t g0 = a.bases[t] + lo_w;
  uint16_t* w = a.ptrs[t] + lo_w;
  const bool vec = len == (uint64_t)kMergeTile && ((uintptr_t)w & 15) == 0;
  mg_u32x4 x[kMergeVec];
  if (vec) {
#pragma unroll
    for (int j = 0; j < kMergeVec; ++j)
      x[j] = __builtin_nontemporal_load((const mg_gv4*)w + threadIdx.x + kApplyThreads * j);
  }
  if (wave < 2) {
    const uint64_t r = wave_lower_bound(a.idx, 0, a.count, (int64_t)(g0 + (wave ? len : 0)));
    if (lane == 0) s_r[wave] = r;
  }
  if (vec) {
#pragma unroll
    for (int j = 0; j < kMergeVec; ++j) ((mg_u32x4*)s_w)[threadIdx.x + kApplyThreads * j] = x[j];
  } else {
    for (uint32_t i = threadIdx.x; i < (uint32_t)len; i += kApplyThreads)
      s_w[i] = gview((const uint16_t*)w)[i];
  }
  __syncthreads();
  const uint64_t e0 = s_r[0], e1 = s_r[1];
  bool bad = false;
  // entries below the first word or past the last of the tensor list
  if (threadIdx.x == 0 && ((b == 0 && e0 > 0) || (b + 1 == a.tiles && e1 < a.count))) bad = true;
  for (uint64_t e = e0 + threadIdx.x; e < e1; e += kApplyThreads * kMergeLoads) {
    int64_t i[kMergeLoads];
    uint16_t v[kMergeLoads];
#pragma unroll
    for (int u = 0; u < kMergeLoads; ++u) {
      const uint64_t k = e + kApplyThreads * u;
      i[u] = k < e1 ? gview(a.idx)[k] : 0;
      v[u] = k < e1 ? gview(a.val)[k] : 0;
    }
#pragma unroll
    for (int u = 0; u < kMergeLoads; ++u) {
      if (e + kApplyThreads * u >= e1) continue;
      const uint64_t o = (uint64_t)i[u] - g0;
      if (o < len)
        s_w[o] = v[u];
      else
        bad = true;   // only out-of-order input puts an entry outside its tile
    }
  }
  __syncthreads();
  if (vec) {
#pragma unroll
    for (int j = 0; j < kMergeVec; ++j)
      __builtin_nontemporal_store(((mg_u32x4*)s_w)[threadIdx.x + kApplyThreads * j],
                                  (mg_gv4*)w + threadIdx.x + kApplyThreads * j);
  } else {
    for (uint32_t i = threadIdx.x; i < (uint32_t)len; i += kApplyThreads)
      ((__attribute__((address_space(1))) uint16_t*)w)[i] = s_w[i];
  }
  if (bad) flag_error(a.err);
}


// ------------------------------------ dense chains: runs of tiles merged
//
// A chain D_1..D_K (oldest first, each strictly increasing) whose entries
// together hold at least one word in 32 of the tensor list: each workgroup
// walks a run of kRunTiles consecutive tiles with one cursor per delta
// (each found once, by a 64-wide search, at the run's first tile).  For a
// tile it loads the tile's words and, beside them, the next chunk of the
// first deltas (L entries per thread per delta, kRunSlots per thread: with
// more than kRunSlots / L deltas the rest follow in batches); then it
// patches the deltas into the tile in LDS oldest first (a
// barrier between deltas, so of equal indices the newest word stays),
// loading further chunks of a delta while its entries still fall in the
// tile, moves every cursor past the entries the tile took, and writes the
// tile back whole.  With K = 1 it is the tile merge of one sorted delta
// without per-tile searches.

constexpr int kRunTiles = 32;   // tiles per workgroup
constexpr int kRunSlots = 8;    // delta entries per thread per batch of deltas

struct RunArgs {
  const uint64_t* bases;
  uint16_t* const* ptrs;
  const uint64_t* tile_first;
  uint32_t T;
  uint64_t tiles;
  const ChainDelta* deltas;   // device [K]
  uint32_t K;
  uint32_t lg;                // chunk loads per thread per delta: L = 2^lg <= kRunSlots
  uint32_t* err;
};

// A value every lane of the wavefront holds alike, in scalar registers.
__device__ __forceinline__ uint64_t run_uniform(uint64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(x >> 32));
  return ((uint64_t)hi << 32) | lo;
}

// Block-wide maximum of v (every thread gets it); one barrier.  Two calls
// in a row must pass different buffers: a wavefront reads the buffer after
// the barrier, and only the next call's barrier orders that read before
// the buffer is written again.
__device__ __forceinline__ uint32_t run_block_max(uint32_t v, uint32_t* s_red) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const uint32_t y = __shfl_xor(v, o);
    v = y > v ? y : v;
  }
  if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6] = v;
  __syncthreads();
  uint32_t m = 0;
#pragma unroll
  for (int w = 0; w < kApplyThreads / 64; ++w) m = s_red[w] > m ? s_red[w] : m;
  return m;
}

__global__ __launch_bounds__(kApplyThreads) void apply_runs_kernel(RunArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t s_w[kMergeTile];
  __shared__ ChainDelta s_d[kChainMaxDeltas];
  __shared__ uint64_t s_cur[kChainMaxDeltas];
  __shared__ uint32_t s_red[2][kApplyThreads / 64];
  __shared__ uint32_t s_t;
  const uint32_t K = a.K, lg = a.lg, L = 1u << lg, chunk = kApplyThreads * L;
  const uint32_t wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const uint64_t b0 = (uint64_t)blockIdx.x * kRunTiles;
  const uint64_t b1 = b0 + kRunTiles < a.tiles ? b0 + kRunTiles : a.tiles;
  bool bad = false;
  if (threadIdx.x < K) s_d[threadIdx.x] = a.deltas[threadIdx.x];
  if (wave == 0) {   // the tensor of tile b0, as in apply_merge_kernel
    uint32_t lo = 0, hi = a.T;
    while (hi - lo > 1) {
      const uint32_t n = hi - lo;
      const uint32_t p = lo + (uint32_t)(((uint64_t)n * lane) >> 6);
      const uint64_t m = __ballot(a.tile_first[p] <= b0);
      const uint32_t c = 63 - (uint32_t)__builtin_clzll(m);
      const uint32_t last = (uint32_t)__shfl((int)p, (int)c);
      const uint32_t next = (uint32_t)__shfl((int)p, (int)(c < 63 ? c + 1 : 63));
      lo = last;
      if (c < 63) hi = next;
    }
    if (lane == 0) s_t = lo;
  }
  __syncthreads();
  uint32_t t = s_t;
  {
    // every delta's cursor at the run's first word: wavefront w searches
    // deltas w, w + 4, ...
    const uint64_t g_first = a.bases[t] + (b0 - a.tile_first[t]) * kMergeTile;
    for (uint32_t k = wave; k < K; k += kApplyThreads / 64) {
      const uint64_t c = wave_lower_bound(s_d[k].idx, 0, s_d[k].n, (int64_t)g_first);
      if (lane == 0) s_cur[k] = c;
    }
  }
  __syncthreads();
  if (b0 == 0 && threadIdx.x < K && s_cur[threadIdx.x] > 0) bad = true;   // entries below word 0
  for (uint64_t b = b0; b < b1; ++b) {
    while (t + 1 < a.T && a.tile_first[t + 1] <= b) ++t;   // uniform
    const uint64_t lo_w = (b - a.tile_first[t]) * kMergeTile;
    const uint64_t n_t = a.bases[t + 1] - a.bases[t];
    const uint64_t len = n_t - lo_w < (uint64_t)kMergeTile ? n_t - lo_w : kMergeTile;
    const uint64_t g0 = a.bases[t] + lo_w;
    const int64_t g_end = (int64_t)(g0 + len);
    uint16_t* w = a.ptrs[t] + lo_w;
    const bool vec = len == (uint64_t)kMergeTile && ((uintptr_t)w & 15) == 0;
    mg_u32x4 x[kMergeVec];
    if (vec) {
#pragma unroll
      for (int j = 0; j < kMergeVec; ++j)
        x[j] = __builtin_nontemporal_load((const mg_gv4*)w + threadIdx.x + kApplyThreads * j);
    }
    // The deltas go in batches of at most kRunSlots >> lg: slot s of a batch
    // starting at delta d0 holds entry cur_k + thread + 256 j of delta
    // k = d0 + (s >> lg), j = s & (L - 1).  The first batch's chunks load
    // beside the tile's words.
    int64_t ei[kRunSlots];
    uint16_t ev[kRunSlots];
    const uint32_t per_batch = kRunSlots >> lg;
    const auto load_batch = [&](uint32_t d0) {
#pragma unroll
      for (int s = 0; s < kRunSlots; ++s) {
        const uint32_t k = d0 + ((uint32_t)s >> lg), j = (uint32_t)s & (L - 1);
        ei[s] = INT64_MAX;
        ev[s] = 0;
        if (k < K && k < d0 + per_batch) {
          const uint64_t cur = run_uniform(s_cur[k]), n = run_uniform(s_d[k].n);
          const int64_t* xi = (const int64_t*)run_uniform((uint64_t)(uintptr_t)s_d[k].idx);
          const uint16_t* xv = (const uint16_t*)run_uniform((uint64_t)(uintptr_t)s_d[k].val);
          const uint64_t e = cur + threadIdx.x + (uint64_t)kApplyThreads * j;
          if (e < n) {
            ei[s] = gview(xi)[e];
            ev[s] = gview(xv)[e];
          }
        }
      }
    };
    load_batch(0);
    if (vec) {
#pragma unroll
      for (int j = 0; j < kMergeVec; ++j) ((mg_u32x4*)s_w)[threadIdx.x + kApplyThreads * j] = x[j];
    } else {
      for (uint32_t i = threadIdx.x; i < (uint32_t)len; i += kApplyThreads)
        s_w[i] = gview((const uint16_t*)w)[i];
    }
    __syncthreads();
    uint32_t red = 0;   // reductions so far: consecutive ones use different buffers
    for (uint32_t d0 = 0; d0 < K; d0 += per_batch) {
      // a later batch: every cursor it reads was published by the barrier
      // of the previous batch's last reduction
      if (d0 > 0) load_batch(d0);
      const uint32_t d1 = d0 + per_batch < K ? d0 + per_batch : K;
      for (uint32_t k = d0; k < d1; ++k) {
        // read before the barrier below, after which thread 0 may move it
        uint64_t cur = run_uniform(s_cur[k]);
        const uint64_t n = run_uniform(s_d[k].n);
        const int64_t* xi = (const int64_t*)run_uniform((uint64_t)(uintptr_t)s_d[k].idx);
        const uint16_t* xv = (const uint16_t*)run_uniform((uint64_t)(uintptr_t)s_d[k].val);
        // this thread's entries of delta k that fall in the tile; the tile
        // takes a prefix of the chunk (sorted input), m = its length
        uint32_t m = 0;
#pragma unroll
        for (int s = 0; s < kRunSlots; ++s) {
          if (d0 + ((uint32_t)s >> lg) != k) continue;
          const uint32_t j = (uint32_t)s & (L - 1);
          // strictly increasing (checked between neighbouring lanes)
          const int64_t nx = __shfl_down(ei[s], 1);
          if (lane != 63 && nx != INT64_MAX && ei[s] != INT64_MAX && nx <= ei[s]) bad = true;
          if (ei[s] < g_end) {
            const uint64_t o = (uint64_t)ei[s] - g0;
            if (o < len)
              s_w[o] = ev[s];
            else
              bad = true;   // below the tile: only unsorted input
            const uint32_t pos = threadIdx.x + kApplyThreads * j + 1;
            m = pos > m ? pos : m;
          }
        }
        m = run_block_max(m, s_red[red++ & 1]);
        // a chunk taken whole: the delta may hold more words of this tile
        while (m == chunk && cur + m < n) {
          cur += m;
          m = 0;
#pragma unroll
          for (int j = 0; j < kRunSlots; ++j) {
            if ((uint32_t)j >= L) break;
            const uint64_t e = cur + threadIdx.x + (uint64_t)kApplyThreads * j;
            if (e < n) {
              const int64_t i = gview(xi)[e];
              if (i < g_end) {
                const uint64_t o = (uint64_t)i - g0;
                if (o < len)
                  s_w[o] = gview(xv)[e];
                else
                  bad = true;
                const uint32_t pos = threadIdx.x + kApplyThreads * j + 1;
                m = pos > m ? pos : m;
              }
            }
          }
          m = run_block_max(m, s_red[red++ & 1]);
        }
        if (threadIdx.x == 0) s_cur[k] = cur + m;
      }
      if (d1 < K) __syncthreads();   // the batch's cursors are published
    }
    __syncthreads();   // the tile is complete; s_cur is published
    if (vec) {
#pragma unroll
      for (int j = 0; j < kMergeVec; ++j)
        __builtin_nontemporal_store(((mg_u32x4*)s_w)[threadIdx.x + kApplyThreads * j],
                                    (mg_gv4*)w + threadIdx.x + kApplyThreads * j);
    } else {
      for (uint32_t i = threadIdx.x; i < (uint32_t)len; i += kApplyThreads)
        ((__attribute__((address_space(1))) uint16_t*)w)[i] = s_w[i];
    }
    __syncthreads();   // s_w is read before the next tile overwrites it
  }
  // entries past the last word
  if (b1 == a.tiles && threadIdx.x < K && s_cur[threadIdx.x] < s_d[threadIdx.x].n) bad = true;
  if (bad) flag_error(a.err);
}

static uint32_t apply_blocks(uint64_t count) {
  const uint64_t per_block = (uint64_t)kApplyWaves * kApplyPerWave;
  uint64_t blocks = (count + per_block - 1) / per_block;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  return (uint32_t)blocks;
}

hipError_t launch_apply(uint16_t* w, uint64_t n, bool idx64, const void* idx,
                        const uint16_t* val, uint64_t count, uint32_t* err,
                        hipStream_t stream) {
  if (count == 0) return hipSuccess;
  if (idx64)
    hipLaunchKernelGGL(apply_kernel<int64_t>, dim3(apply_blocks(count)), dim3(kApplyThreads), 0,
                       stream, w, n, (const int64_t*)idx, val, count, err);
  else
    hipLaunchKernelGGL(apply_kernel<int32_t>, dim3(apply_blocks(count)), dim3(kApplyThreads), 0,
                       stream, w, n, (const int32_t*)idx, val, count, err);
  return hipGetLastError();
}

hipError_t launch_apply_multi(const uint64_t* bases, uint16_t* const* ptrs, uint32_t T,
                              const int64_t* idx, const uint16_t* val, uint64_t count,
                              uint32_t* err, hipStream_t stream) {
  if (count == 0) return hipSuccess;
  hipLaunchKernelGGL(apply_multi_kernel, dim3(apply_blocks(count)), dim3(kApplyThreads), 0, stream,
                     bases, ptrs, T, idx, val, count, err);
  return hipGetLastError();
}


uint64_t merge_tiles(const uint64_t* numels, uint32_t T, uint64_t* tile_first) {
  uint64_t tiles = 0;
  for (uint32_t t = 0; t < T; ++t) {
    if (tile_first) tile_first[t] = tiles;
    tiles += (numels[t] + kMergeTile - 1) / kMergeTile;
  }
  if (tile_first) tile_first[T] = tiles;
  return tiles;
}

bool merge_pays(uint64_t count, uint64_t words) { return count > 0 && count >= words / 32; }

bool chain_merge_pays(uint64_t entries, uint64_t words) {
  return entries > 0 && entries >= words / 24;
}

hipError_t launch_apply_merge(const uint64_t* bases, uint16_t* const* ptrs,
                              const uint64_t* tile_first, uint32_t T, uint64_t tiles,
                              const int64_t* idx, const uint16_t* val, uint64_t count,
                              uint32_t* err, hipStream_t stream) {
  if (tiles == 0) return hipSuccess;
  MergeArgs a{bases, ptrs, tile_first, T, tiles, idx, val, count, err};
  hipLaunchKernelGGL(apply_merge_kernel, dim3((uint32_t)tiles), dim3(kApplyThreads), 0, stream,
                     a);
  return hipGetLastError();
}


hipError_t launch_apply_runs(const uint64_t* bases, uint16_t* const* ptrs,
                             const uint64_t* tile_first, uint32_t T, uint64_t tiles,
                             const ChainDelta* deltas, uint32_t K, uint64_t entries,
                             uint64_t words, uint32_t* err, hipStream_t stream) {
  if (tiles == 0 || K == 0) return hipSuccess;
  // chunk loads per thread per delta: the entries an average tile holds of
  // the average delta, with room, within the slots
  const uint64_t per_tile = entries / K * kMergeTile / (words ? words : 1);
  const uint64_t want = (per_tile * 5 / 4 + kApplyThreads - 1) / kApplyThreads;
  uint32_t lg = 0;   // the smallest power of two >= want that one batch of all deltas allows
  while ((1ull << lg) < want && (K << (lg + 1)) <= (uint32_t)kRunSlots) ++lg;
  RunArgs a{bases, ptrs, tile_first, T, tiles, deltas, K, lg, err};
  const uint64_t runs = (tiles + kRunTiles - 1) / kRunTiles;
  hipLaunchKernelGGL(apply_runs_kernel, dim3((uint32_t)runs), dim3(kApplyThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace aurora
