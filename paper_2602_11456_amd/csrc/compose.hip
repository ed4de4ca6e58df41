// Delta chain composition on gfx950 (AuroraRL Sec. 5.4, "Version-predicate
// join and delta catch-up"): a worker K versions behind replays the missed
// deltas in order.  Apply assigns, so the chain equals one delta holding
// every index of the chain with the value of the newest delta that has it.
//
// Two deltas A (older) and B (newer) merge with a merge path (Green,
// McColl and Bader, "GPU merge path", 2012): workgroup t takes the merged
// positions [4096 t, 4096 t + 4096); where every tile starts in A and B is
// found first by one binary search on the diagonal per tile boundary (one
// thread each), the workgroup stages both pieces in LDS, and each thread
// merges 16 positions.  Ties put A first; an A entry whose
// index B also holds is dropped (B's value wins).  A count pass, the group
// scan of the per-tile counts, and a write pass give the compacted output.
// Longer chains merge pairwise in rounds (a tree), with every count kept
// on the device, so a whole composition is enqueued without a host wait.
#include <string.h>

#include <vector>

#include "delta_internal.h"

namespace aurora {

constexpr int kCmpThreads = 256;
constexpr int kCmpPer = 16;                          // merged positions per thread
constexpr int kCmpTile = kCmpThreads * kCmpPer;      // 4096
constexpr int kCmpLoad = 8;                          // staging loads in flight per thread

struct ComposeArgs {
  const int64_t* a_idx;
  const uint16_t* a_val;
  uint64_t na;             // entries of A, or the most there can be if d_na is set
  const uint64_t* d_na;    // nullable: A's count in device memory
  const int64_t* b_idx;
  const uint16_t* b_val;
  uint64_t nb;
  const uint64_t* d_nb;
  int64_t* out_idx;
  uint16_t* out_val;
  uint64_t capacity;
  uint32_t* tile_counts;
  uint64_t* group_excl;
  uint64_t* splits;        // entries of A before each tile boundary (tiles + 1)
  uint32_t* err;           // nullable: set when the merge meets unsorted input
};

__device__ __forceinline__ uint64_t live_count(uint64_t n, const uint64_t* d_n) {
  if (!d_n) return n;
  const uint64_t c = *d_n;
  return c < n ? c : n;
}

// Merged position d -> entries of A before it (ties: A first).  Always in
// [max(0, d - nb), min(d, na)].
template <typename GetA, typename GetB>
__device__ __forceinline__ uint64_t diag_split(GetA A, GetB B, uint64_t na, uint64_t nb,
                                               uint64_t d) {
  uint64_t lo = d > nb ? d - nb : 0, hi = d < na ? d : na;
  while (lo < hi) {
    const uint64_t mid = (lo + hi) >> 1;
    if (A(mid) <= B(d - mid - 1)) lo = mid + 1; else hi = mid;
  }
  return lo;
}

// splits[b] = entries of A before merged position min(b * kCmpTile, na + nb),
// one thread per tile boundary.
__global__ void compose_split_kernel(ComposeArgs a, uint64_t num_bounds) {
  const uint64_t b = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= num_bounds) return;
  const uint64_t na = live_count(a.na, a.d_na), nb = live_count(a.nb, a.d_nb);
  const uint64_t total = na + nb;
  const uint64_t d = b * kCmpTile < total ? b * kCmpTile : total;
  auto A = [&](uint64_t i) { return a.a_idx[i]; };
  auto B = [&](uint64_t j) { return a.b_idx[j]; };
  a.splits[b] = diag_split(A, B, na, nb, d);
}

// One tile of the merge: its bounds in A and B, staged in LDS.
struct CmpTile {
  uint64_t i0, j0;      // first entries of A and B in the tile
  uint32_t la, lb;      // entries of A and B in the tile
  uint32_t positions;   // merged positions of the tile
  bool ext;             // s_b[lb] holds B's next entry (for the duplicate test)
  bool ok;
};

// Block-wide (a barrier after the staging).  Returns ok = false for a tile
// past the end or for inconsistent (unsorted) input.
__device__ __forceinline__ CmpTile cmp_load_tile(const ComposeArgs& a, uint64_t tile,
                                                 uint64_t na, uint64_t nb, int64_t* s_ab) {
  CmpTile t{};
  const uint64_t d0 = tile * kCmpTile;
  const uint64_t total = na + nb;
  if (d0 >= total) return t;   // uniform
  const uint64_t d1 = d0 + kCmpTile < total ? d0 + kCmpTile : total;
  const uint64_t i0 = a.splits[tile], i1 = a.splits[tile + 1];
  const uint64_t j0 = d0 - i0, j1 = d1 - i1;
  if (i1 < i0 || j1 < j0 || i0 > d0 || i1 > d1) {   // only unsorted input gets here
    if (threadIdx.x == 0 && a.err)
      __hip_atomic_fetch_or(a.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return t;
  }
  t.i0 = i0;
  t.j0 = j0;
  t.la = (uint32_t)(i1 - i0);
  t.lb = (uint32_t)(j1 - j0);
  t.positions = (uint32_t)(d1 - d0);
  t.ext = j1 < nb;
  const uint32_t nload = t.la + t.lb + (t.ext ? 1u : 0u);
  // kCmpLoad loads per thread in flight before any LDS store
  for (uint32_t q0 = 0; q0 < nload; q0 += kCmpThreads * kCmpLoad) {
    int64_t v[kCmpLoad];
#pragma unroll
    for (int k = 0; k < kCmpLoad; ++k) {
      const uint32_t q = q0 + threadIdx.x + kCmpThreads * k;
      v[k] = q < nload ? (q < t.la ? a.a_idx[i0 + q] : a.b_idx[j0 + (q - t.la)]) : 0;
    }
#pragma unroll
    for (int k = 0; k < kCmpLoad; ++k) {
      const uint32_t q = q0 + threadIdx.x + kCmpThreads * k;
      if (q < nload) s_ab[q] = v[k];
    }
  }
  __syncthreads();
  t.ok = true;
  return t;
}

// Walks this thread's merged positions; emit(index, from_b, position in
// its tile piece) is called for every kept entry, in order.
template <typename Emit>
__device__ __forceinline__ void cmp_walk(const CmpTile& t, const int64_t* s_ab, uint64_t nb,
                                         Emit emit) {
  const int64_t* sA = s_ab;
  const int64_t* sB = s_ab + t.la;
  const uint32_t p0 = threadIdx.x * kCmpPer;
  if (p0 >= t.positions) return;
  uint32_t lo = p0 > t.lb ? p0 - t.lb : 0, hi = p0 < t.la ? p0 : t.la;
  while (lo < hi) {
    const uint32_t mid = (lo + hi) >> 1;
    if (sA[mid] <= sB[p0 - mid - 1]) lo = mid + 1; else hi = mid;
  }
  uint32_t i = lo, j = p0 - lo;
  const uint32_t n = t.positions - p0 < (uint32_t)kCmpPer ? t.positions - p0 : kCmpPer;
  for (uint32_t s = 0; s < n; ++s) {
    if (i < t.la && (j >= t.lb || sA[i] <= sB[j])) {
      // dropped when B holds the same index (it comes right after)
      const bool dup = t.j0 + j < nb && (j < t.lb || t.ext) && sB[j] == sA[i];
      if (!dup) emit(sA[i], false, i);
      ++i;
    } else {
      emit(sB[j], true, j);
      ++j;
    }
  }
}

__device__ __forceinline__ uint32_t cmp_block_sum(uint32_t v, uint32_t* s_wave) {
  uint32_t x = v;
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) x += __shfl_xor(x, s);
  if ((threadIdx.x & 63) == 0) s_wave[threadIdx.x >> 6] = x;
  __syncthreads();
  uint32_t t = 0;
  for (int w = 0; w < kCmpThreads / 64; ++w) t += s_wave[w];
  __syncthreads();
  return t;
}

__global__ __launch_bounds__(kCmpThreads) void compose_count_kernel(ComposeArgs a) {
  __shared__ int64_t s_ab[kCmpTile + 1];
  __shared__ uint32_t s_wave[kCmpThreads / 64];
  const uint64_t na = live_count(a.na, a.d_na), nb = live_count(a.nb, a.d_nb);
  const CmpTile t = cmp_load_tile(a, blockIdx.x, na, nb, s_ab);
  uint32_t kept = 0;
  if (t.ok) cmp_walk(t, s_ab, nb, [&](int64_t, bool, uint32_t) { ++kept; });
  const uint32_t total = cmp_block_sum(kept, s_wave);
  if (threadIdx.x == 0) a.tile_counts[blockIdx.x] = total;
}

// Write pass: the walk keeps each thread's merged entries in registers, the
// tile's kept entries are assembled in LDS (over the staged input), and the
// workgroup stores them as one contiguous, coalesced run.
__global__ __launch_bounds__(kCmpThreads) void compose_write_kernel(ComposeArgs a) {
  __shared__ int64_t s_ab[kCmpTile + 1];
  __shared__ uint16_t s_vab[kCmpTile];
  __shared__ uint32_t s_wave[kCmpThreads / 64];
  __shared__ uint64_t s_before;
  const uint64_t na = live_count(a.na, a.d_na), nb = live_count(a.nb, a.d_nb);
  const uint64_t tile = blockIdx.x;
  const CmpTile t = cmp_load_tile(a, tile, na, nb, s_ab);
  if (!t.ok) return;   // uniform
  for (uint32_t q0 = 0; q0 < t.la + t.lb; q0 += kCmpThreads * kCmpLoad) {
    uint16_t v[kCmpLoad];
#pragma unroll
    for (int k = 0; k < kCmpLoad; ++k) {
      const uint32_t q = q0 + threadIdx.x + kCmpThreads * k;
      v[k] = q < t.la + t.lb ? (q < t.la ? a.a_val[t.i0 + q] : a.b_val[t.j0 + (q - t.la)]) : 0;
    }
#pragma unroll
    for (int k = 0; k < kCmpLoad; ++k) {
      const uint32_t q = q0 + threadIdx.x + kCmpThreads * k;
      if (q < t.la + t.lb) s_vab[q] = v[k];
    }
  }
  __syncthreads();
  // merged position s of this thread: oi[s], ov[s]; bit s of keep: kept
  int64_t oi[kCmpPer];
  uint16_t ov[kCmpPer];
  uint32_t keep = 0;
  {
    const int64_t* sA = s_ab;
    const int64_t* sB = s_ab + t.la;
    const uint32_t p0 = threadIdx.x * kCmpPer;
    uint32_t i = 0, j = 0, n = 0;
    if (p0 < t.positions) {
      uint32_t lo = p0 > t.lb ? p0 - t.lb : 0, hi = p0 < t.la ? p0 : t.la;
      while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        if (sA[mid] <= sB[p0 - mid - 1]) lo = mid + 1; else hi = mid;
      }
      i = lo;
      j = p0 - lo;
      n = t.positions - p0 < (uint32_t)kCmpPer ? t.positions - p0 : kCmpPer;
    }
#pragma unroll
    for (uint32_t s = 0; s < (uint32_t)kCmpPer; ++s) {
      oi[s] = 0;
      ov[s] = 0;
      if (s < n) {
        if (i < t.la && (j >= t.lb || sA[i] <= sB[j])) {
          // dropped when B holds the same index (it comes right after)
          const bool dup = (j < t.lb || t.ext) && sB[j] == sA[i];
          oi[s] = sA[i];
          ov[s] = s_vab[i];
          keep |= (uint32_t)!dup << s;
          ++i;
        } else {
          oi[s] = sB[j];
          ov[s] = s_vab[t.la + j];
          keep |= 1u << s;
          ++j;
        }
      }
    }
  }
  const uint32_t kept = __builtin_popcount(keep);
  // exclusive prefix of `kept` over the workgroup
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t x = kept;
#pragma unroll
  for (int s = 1; s < 64; s <<= 1) {
    const uint32_t y = __shfl_up(x, s);
    if ((int)lane >= s) x += y;
  }
  if (lane == 63) s_wave[wave] = x;
  if (threadIdx.x < 64) {   // kept entries of the group's tiles before this one
    const uint64_t g0 = tile / kTilesPerGroup * kTilesPerGroup;
    uint64_t c = g0 + threadIdx.x < tile ? (uint64_t)a.tile_counts[g0 + threadIdx.x] : 0;
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) c += __shfl_xor(c, s);
    if (threadIdx.x == 0) s_before = c;
  }
  __syncthreads();   // also: every thread is done reading the staged input
  uint32_t local = x - kept;
  uint32_t tile_kept = 0;
  for (int w = 0; w < kCmpThreads / 64; ++w) {
    if (w < (int)wave) local += s_wave[w];
    tile_kept += s_wave[w];
  }
#pragma unroll
  for (uint32_t s = 0; s < (uint32_t)kCmpPer; ++s) {
    if ((keep >> s) & 1u) {
      s_ab[local] = oi[s];
      s_vab[local] = ov[s];
      ++local;
    }
  }
  __syncthreads();
  const uint64_t base = a.group_excl[tile / kTilesPerGroup] + s_before;
  for (uint32_t q = threadIdx.x; q < tile_kept; q += kCmpThreads) {
    if (base + q < a.capacity) {
      a.out_idx[base + q] = s_ab[q];
      a.out_val[base + q] = s_vab[q];
    }
  }
}

static uint64_t cmp_tiles(uint64_t n) { return (n + kCmpTile - 1) / kCmpTile; }

// Scratch of one pairwise merge of up to n merged positions.
struct CmpScratch {
  size_t tile_counts, group_sum, group_excl, splits, total;
};
static CmpScratch cmp_scratch(uint64_t n) {
  CmpScratch s;
  const uint64_t tiles = cmp_tiles(n), groups = groups_for(tiles);
  s.tile_counts = 0;
  s.group_sum = align_up(4 * tiles);
  s.group_excl = align_up(s.group_sum + 8 * groups);
  s.splits = align_up(s.group_excl + 8 * groups);
  s.total = align_up(s.splits + 8 * (tiles + 1));
  return s;
}

static hipError_t launch_compose2(ComposeArgs a, char* scratch, uint64_t* d_count,
                                  hipStream_t stream) {
  const uint64_t tiles = cmp_tiles(a.na + a.nb);
  if (tiles == 0) return launch_reset(d_count, nullptr, 0, stream);
  const CmpScratch s = cmp_scratch(a.na + a.nb);
  a.tile_counts = (uint32_t*)(scratch + s.tile_counts);
  a.group_excl = (uint64_t*)(scratch + s.group_excl);
  a.splits = (uint64_t*)(scratch + s.splits);
  const uint64_t bounds = tiles + 1;
  hipLaunchKernelGGL(compose_split_kernel, dim3((uint32_t)((bounds + 255) / 256)), dim3(256), 0,
                     stream, a, bounds);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(compose_count_kernel, dim3((uint32_t)tiles), dim3(kCmpThreads), 0, stream, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = launch_group_scan(a.tile_counts, tiles, (uint64_t*)(scratch + s.group_sum), a.group_excl,
                        d_count, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(compose_write_kernel, dim3((uint32_t)tiles), dim3(kCmpThreads), 0, stream, a);
  return hipGetLastError();
}

// ------------------------------------------------------------ the chain

// Workspace: scratch of the largest merge, one count slot per delta, and
// the intermediate results of every round but the last (each round's
// results together hold at most `total` entries).
ChainLayout chain_layout(const uint64_t* counts, int32_t K) {
  ChainLayout L;
  uint64_t total = 0;
  for (int32_t d = 0; d < K; ++d) total += counts[d];
  uint64_t rounds = 0;
  for (int64_t items = K; items > 1; items = (items + 1) / 2) ++rounds;
  if (K == 1) rounds = 1;   // one merge with an empty delta: a copy
  L.rounds = rounds;
  L.scratch = 0;
  L.counts = align_up(cmp_scratch(total).total);
  L.inter = align_up(L.counts + 8 * (uint64_t)(K > 0 ? K : 1));
  const uint64_t inter_rounds = rounds > 1 ? rounds - 1 : 0;
  L.total = align_up(L.inter + inter_rounds * (align_up(8 * total) + align_up(2 * total)));
  return L;
}

hipError_t launch_compose_chain(const int64_t* const* idx, const uint16_t* const* val,
                                const uint64_t* counts, int32_t K, int64_t* out_idx,
                                uint16_t* out_val, uint64_t capacity, uint64_t* d_count,
                                uint32_t* err, char* ws, hipStream_t stream) {
  if (K == 0) return launch_reset(d_count, nullptr, 0, stream);
  const ChainLayout L = chain_layout(counts, K);
  uint64_t total = 0;
  for (int32_t d = 0; d < K; ++d) total += counts[d];
  struct Item {
    const int64_t* idx;
    const uint16_t* val;
    uint64_t ub;            // at most this many entries
    const uint64_t* d_n;    // its count on the device (NULL: exactly ub)
  };
  std::vector<Item> items;
  for (int32_t d = 0; d < K; ++d) items.push_back({idx[d], val[d], counts[d], nullptr});
  if (K == 1) items.push_back({nullptr, nullptr, 0, nullptr});
  uint64_t* slots = (uint64_t*)(ws + L.counts);
  uint32_t slot = 0;
  uint64_t round = 0;
  while (items.size() > 1) {
    const bool last = items.size() == 2;
    char* region = ws + L.inter + round * (align_up(8 * total) + align_up(2 * total));
    int64_t* r_idx = (int64_t*)region;
    uint16_t* r_val = (uint16_t*)(region + align_up(8 * total));
    uint64_t r_off = 0;
    std::vector<Item> next;
    for (size_t p = 0; p + 1 < items.size(); p += 2) {
      const Item& x = items[p];
      const Item& y = items[p + 1];
      ComposeArgs a;
      memset(&a, 0, sizeof(a));
      a.a_idx = x.idx;
      a.a_val = x.val;
      a.na = x.ub;
      a.d_na = x.d_n;
      a.b_idx = y.idx;
      a.b_val = y.val;
      a.nb = y.ub;
      a.d_nb = y.d_n;
      a.err = err;
      uint64_t* cnt;
      if (last) {
        a.out_idx = out_idx;
        a.out_val = out_val;
        a.capacity = capacity;
        cnt = d_count;
      } else {
        a.out_idx = r_idx + r_off;
        a.out_val = r_val + r_off;
        a.capacity = x.ub + y.ub;
        cnt = slots + slot++;
      }
      hipError_t e = launch_compose2(a, ws + L.scratch, cnt, stream);
      if (e != hipSuccess) return e;
      next.push_back({a.out_idx, a.out_val, x.ub + y.ub, cnt});
      r_off += x.ub + y.ub;
    }
    if (items.size() % 2) next.push_back(items.back());
    items.swap(next);
    ++round;
  }
  return hipSuccess;
}

}  // namespace aurora
