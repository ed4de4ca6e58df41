// Sparse delta extraction on gfx950: keep every bf16 word whose bits
// changed between the two copies and write the kept positions and new
// words, in ascending position order, as two dense streams (AuroraRL
// Sec. 5.1, "Sparse encoding").
//
// The word space is cut into tiles of 8192 words (tiles never span
// tensors).  Three kernels:
//
//   stage     One workgroup per tile streams both copies once (16-byte
//             loads, 8 words per lane per load), compares 16-bit words,
//             turns per-lane change counts into lane prefixes with four
//             ballots + mbcnt (a bit-sliced prefix sum), combines the
//             wavefront totals through LDS, and writes the tile's kept
//             entries, in order, into the tile's own staging slot, plus the
//             tile's count.  No workgroup ever waits on another.
//   scan      Per-group (64 tiles) sums, then one workgroup scans the group
//             sums: every group's output offset and the grand total.
//   finalize  One workgroup per group scans its 64 tile counts and copies
//             each tile's staged entries to their final positions as
//             global indices.  A tile with more kept words than its slot
//             holds is read again here and written directly.
//
// Why not a single pass with a decoupled look-back (Merrill & Garland,
// 2016): there a tile can write only after every earlier tile has
// published its count, i.e. after their loads have returned, and the
// jitter of HBM load completion then stalls whole convoys of workgroups
// with nothing in flight.  Measured on this part that ran at about half of
// the read ceiling, while this split reaches it.  The price is writing and
// re-reading the staged entries: 8 bytes per kept word, about 2% extra
// traffic at 1% density.
#include "delta_internal.h"

namespace aurora {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(1))) u32x4* gvec_ptr;

__device__ __forceinline__ uint32_t lane_id() {
  return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
}

// Number of set bits of `mask` in lanes below this one.
__device__ __forceinline__ uint32_t mbcnt64(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ uint64_t wave_sum64(uint64_t v) {
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) v += __shfl_xor(v, s);
  return v;
}

// Loads group g (words 8g - head .. 8g - head + 7 of the slice) of both
// copies and returns which of its 8 words lie inside the slice.
//
// kVec (prev and next share their alignment): the group is one aligned
// 16-byte chunk of each copy.  An edge group is read whole as well: a
// 16-byte aligned chunk that holds a word of the slice lies in a page of
// the slice's allocation, so the read cannot fault; the words outside the
// slice are masked off.  !kVec (copies aligned differently, a rare layout
// with kernel instances of its own): the group is read word by word.
template <bool kVec>
__device__ __forceinline__ uint32_t load_group(const TensorDesc& d, int64_t g, u32x4& p,
                                               u32x4& q) {
  const int64_t e0 = 8 * g - (int64_t)d.head;
  const int64_t lo = e0 < 0 ? -e0 : 0;
  const int64_t hi = (int64_t)d.n - e0 < 8 ? (int64_t)d.n - e0 : 8;
  if (hi <= lo) {
    p = u32x4{0, 0, 0, 0};
    q = p;
    return 0;
  }
  const uint32_t valid = (0xFFu >> (8 - hi)) & (0xFFu << lo);
  if (kVec) {
    const gvec_ptr pp = (gvec_ptr)(reinterpret_cast<uintptr_t>(d.prev) - 2u * d.head) + g;
    const gvec_ptr qq = (gvec_ptr)(reinterpret_cast<uintptr_t>(d.next) - 2u * d.head) + g;
    p = __builtin_nontemporal_load(pp);
    q = __builtin_nontemporal_load(qq);
  } else {
    uint32_t pw[4] = {0, 0, 0, 0}, qw[4] = {0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if ((valid >> j) & 1u) {
        pw[j >> 1] |= (uint32_t)d.prev[e0 + j] << (16 * (j & 1));
        qw[j >> 1] |= (uint32_t)d.next[e0 + j] << (16 * (j & 1));
      }
    }
    p = u32x4{pw[0], pw[1], pw[2], pw[3]};
    q = u32x4{qw[0], qw[1], qw[2], qw[3]};
  }
  return valid;
}

// Per 16-bit half of x: 1 if the half is nonzero, else 0 (packed unsigned
// minimum with 1; one instruction for both halves).
__device__ __forceinline__ uint32_t nonzero_halves(uint32_t x) {
  uint32_t r;
  asm("v_pk_min_u16 %0, %1, %2" : "=v"(r) : "v"(x), "s"(0x00010001u));
  return r;
}

// Bit j of the result is set when word j of the group changed.  The two
// flags of dword d sit at bits 0 and 16 of nonzero_halves(p[d] ^ q[d]);
// they are packed to bits 2d and 2d + 1.
__device__ __forceinline__ uint32_t changed_mask(const u32x4& p, const u32x4& q) {
  const uint32_t r0 = nonzero_halves(p[0] ^ q[0]), r1 = nonzero_halves(p[1] ^ q[1]);
  const uint32_t r2 = nonzero_halves(p[2] ^ q[2]), r3 = nonzero_halves(p[3] ^ q[3]);
  const uint32_t s = (r0 | (r1 << 2)) | ((r2 | (r3 << 2)) << 4);   // low flags at 0,2,4,6; high at 16..22
  return (s & 0x55u) | (s >> 15);
}

// Word j (0..7) of a group.
__device__ __forceinline__ uint16_t word_of(const u32x4& q, int j) {
  const uint64_t lo = ((uint64_t)q[1] << 32) | q[0];
  const uint64_t hi = ((uint64_t)q[3] << 32) | q[2];
  return (uint16_t)(((j & 4) ? hi : lo) >> (16 * (j & 3)));
}

// Row of the inline slice holding `tile`: the last whose first tile is at
// or below it.
__device__ __forceinline__ uint32_t inline_row(const ExtractArgs& a, uint64_t tile) {
  uint32_t r = 0;
#pragma unroll
  for (int k = 1; k < kInlineDescs; ++k)   // unrolled: all loads issue at once
    r = ((uint32_t)k < a.num_inline && tile >= a.inl[k].first_tile) ? (uint32_t)k : r;
  return r;
}

// Descriptor of the slice holding `tile`.  The tile id is uniform across
// the wavefront, so every field is moved to scalar registers.
template <bool kMulti>
__device__ __forceinline__ TensorDesc tile_desc(const ExtractArgs& a, uint64_t tile) {
  if (!kMulti) return a.inl[__builtin_amdgcn_readfirstlane(inline_row(a, tile))];
  const uint32_t row = __builtin_amdgcn_readfirstlane(a.tile_map[tile]);
  const uint32_t* src = reinterpret_cast<const uint32_t*>(a.table + row);
  TensorDesc d;
  uint32_t* dst = reinterpret_cast<uint32_t*>(&d);
#pragma unroll
  for (int i = 0; i < (int)(sizeof(TensorDesc) / 4); ++i)
    dst[i] = __builtin_amdgcn_readfirstlane(src[i]);
  return d;
}

// Output index of word 0 of `tile`: the slice base plus the slice word
// index, which is negative inside a misaligned head.
__device__ __forceinline__ int64_t tile_out_base(const TensorDesc& d, uint64_t tile) {
  return (int64_t)d.base + (int64_t)((tile - d.first_tile) * kElemsPerTile) - (int64_t)d.head;
}

// Per-lane result of comparing one tile: which words changed, where they go
// inside the tile's run, and the run length.
struct TileScan {
  u32x4 q[kChunks];               // new words
  uint32_t mask[kChunks];         // bit j: word j of the lane's group changed
  uint32_t rank[kChunks];         // position in the tile's run of the lane's first kept word
  uint32_t tile_total;
};

// Reads and compares one tile with the whole workgroup (kWaves wavefronts).
// Wave w handles groups [w * kGroupsPerWave, (w + 1) * kGroupsPerWave) of
// the tile, chunk u of it being the 64 groups lane + 64u.
template <bool kVec>
__device__ __forceinline__ void scan_tile(const TensorDesc& d, uint64_t tile, uint32_t lane,
                                          uint32_t wave, uint32_t* s_wave_total, TileScan& s) {
  const uint32_t lane_group = wave * kGroupsPerWave + lane;
  const int64_t g0 = (int64_t)((tile - d.first_tile) * kGroupsPerTile) + lane_group;
  const int64_t tile_e0 = (int64_t)((tile - d.first_tile) * kElemsPerTile) - (int64_t)d.head;
  u32x4 p[kChunks];
  if (kVec && tile_e0 >= 0 && tile_e0 + kElemsPerTile <= (int64_t)d.n) {
    // interior tile (almost all of them): no per-group bounds
    const gvec_ptr pp = (gvec_ptr)(reinterpret_cast<uintptr_t>(d.prev) - 2u * d.head) + g0;
    const gvec_ptr qq = (gvec_ptr)(reinterpret_cast<uintptr_t>(d.next) - 2u * d.head) + g0;
#pragma unroll
    for (int u = 0; u < kChunks; ++u) {
      p[u] = __builtin_nontemporal_load(pp + 64 * u);
      s.q[u] = __builtin_nontemporal_load(qq + 64 * u);
    }
#pragma unroll
    for (int u = 0; u < kChunks; ++u) s.mask[u] = changed_mask(p[u], s.q[u]);
  } else {
#pragma unroll
    for (int u = 0; u < kChunks; ++u) {
      const uint32_t valid = load_group<kVec>(d, g0 + 64 * u, p[u], s.q[u]);
      s.mask[u] = changed_mask(p[u], s.q[u]) & valid;
    }
  }
  uint32_t wave_total = 0;
#pragma unroll
  for (int u = 0; u < kChunks; ++u) {
    // Prefix sum of the per-lane counts (0..8) over the wavefront.  When
    // no lane has two or more, one ballot and mbcnt give it; otherwise a
    // bit-sliced sum over the four count bits.
    const uint32_t c = __popc(s.mask[u]);
    const uint64_t any = __ballot(c != 0);
    if (__ballot(c > 1) == 0) {
      s.rank[u] = wave_total + mbcnt64(any);
      wave_total += __popcll(any);
    } else {
      const uint64_t b0 = __ballot(c & 1), b1 = __ballot(c & 2);
      const uint64_t b2 = __ballot(c & 4), b3 = __ballot(c & 8);
      s.rank[u] = wave_total + mbcnt64(b0) + 2 * mbcnt64(b1) + 4 * mbcnt64(b2) + 8 * mbcnt64(b3);
      wave_total += __popcll(b0) + 2 * __popcll(b1) + 4 * __popcll(b2) + 8 * __popcll(b3);
    }
  }
  if (lane == 0) s_wave_total[wave] = wave_total;
  __syncthreads();
  uint32_t wave_excl = 0, total = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const uint32_t t = s_wave_total[w];
    wave_excl += (w < (int)wave) ? t : 0u;
    total += t;
  }
#pragma unroll
  for (int u = 0; u < kChunks; ++u) s.rank[u] += wave_excl;
  s.tile_total = total;
}

// ---------------------------------------------------------------- stage

static_assert(kLdsStage >= kElemsPerTile, "the LDS staging area holds a whole tile");

// Record a coded tile leaves in place of its count, in one 8-byte store:
// kept words (bits 0-13), code bytes of the gaps between consecutive kept
// words (14-27; each gap is below 8192, so one or two bytes), and the tile
// offsets of the first (28-40) and last (41-53) kept word.
static_assert(kElemsPerTile <= 8192, "tile record field widths");
__device__ __forceinline__ uint64_t tile_record(uint32_t count, uint32_t inner, uint32_t first,
                                                uint32_t last) {
  return (uint64_t)count | ((uint64_t)inner << 14) | ((uint64_t)first << 28) |
         ((uint64_t)last << 41);
}
__device__ __forceinline__ uint32_t rec_count(uint64_t r) { return (uint32_t)(r & 0x3FFFu); }
__device__ __forceinline__ uint32_t rec_inner(uint64_t r) { return (uint32_t)((r >> 14) & 0x3FFFu); }
__device__ __forceinline__ uint32_t rec_first(uint64_t r) { return (uint32_t)((r >> 28) & 0x1FFFu); }
__device__ __forceinline__ uint32_t rec_last(uint64_t r) { return (uint32_t)((r >> 41) & 0x1FFFu); }

// kCoded (the coded output of launch_extract_coded): the LDS area holds
// every entry of the tile, and the tile leaves its record (above) instead
// of its count; wavefront 0 sums the gaps' code bytes.

// The dispatcher hands workgroup b to XCD b % 8.  With tile b for workgroup
// b, neighbouring tiles (and the HBM pages they read) go to different XCDs;
// this order gives XCD x a contiguous eighth of the tiles instead (measured
// 4.5% faster for the stage kernel on 8.19 G words).  A bijection of
// [0, tiles).
__device__ __forceinline__ uint64_t xcd_tile(uint64_t b, uint64_t tiles) {
  const uint64_t x = b % 8, q = b / 8, per = tiles / 8, rem = tiles % 8;
  return x * per + (x < rem ? x : rem) + q;
}

template <bool kMulti, bool kVec, bool kCoded>
__global__ __launch_bounds__(kThreads) void stage_kernel(ExtractArgs a) {
  __shared__ uint32_t s_wave_total[kWaves];
  __shared__ __attribute__((aligned(16))) uint32_t s_stage[kLdsStage];
  const uint64_t tile = xcd_tile(blockIdx.x, a.num_tiles);
  const uint32_t lane = lane_id();
  const uint32_t wave = threadIdx.x >> 6;
  const TensorDesc d = tile_desc<kMulti>(a, tile);
  TileScan s;
  scan_tile<kVec>(d, tile, lane, wave, s_wave_total, s);
  // staged entry: (new word << 16) | word offset in the tile
  uint32_t* slot = a.stage + tile * a.stage_stride;
  const uint32_t lane_word = (wave * kGroupsPerWave + lane) * 8;
  const uint32_t keep = s.tile_total < a.stage_cap ? s.tile_total : a.stage_cap;
  const uint32_t in_lds = kCoded ? s.tile_total : keep;
  // Entries go through LDS (which holds a whole tile) so that the slot is
  // written with contiguous stores.
#pragma unroll
  for (int u = 0; u < kChunks; ++u) {
    uint32_t m = s.mask[u];
    uint32_t r = s.rank[u];
    const uint32_t w0 = lane_word + 512 * u;
    while (m) {
      const int j = __builtin_ctz(m);
      m &= m - 1;
      if (r < in_lds) s_stage[r] = ((uint32_t)word_of(s.q[u], j) << 16) | (w0 + j);
      ++r;
    }
  }
  __syncthreads();
  // Streaming (non-temporal) stores: the slot is read once, by another
  // kernel, so it should not displace anything in the caches.
  for (uint32_t r = threadIdx.x; r < keep; r += kThreads)
    __builtin_nontemporal_store(s_stage[r], slot + r);
  if (kCoded) {
    if (wave == 0) {
      uint32_t bytes = 0;
      for (uint32_t r = lane + 1; r < s.tile_total; r += 64) {
        const uint32_t gap = (s_stage[r] & 0xFFFFu) - (s_stage[r - 1] & 0xFFFFu);
        bytes += gap < 128u ? 1u : 2u;
      }
#pragma unroll
      for (int sh = 32; sh >= 1; sh >>= 1) bytes += __shfl_xor(bytes, sh);
      if (lane == 0) {
        const uint32_t n = s.tile_total;
        a.tile_rec[tile] = tile_record(n, bytes, n ? (s_stage[0] & 0xFFFFu) : 0u,
                                       n ? (s_stage[n - 1] & 0xFFFFu) : 0u);
      }
    }
  } else if (threadIdx.x == 0) {
    a.counts[tile] = s.tile_total;
  }
}

// Count only: the same reads and compares as the stage kernel, and only
// the tile's count leaves the workgroup.  The launch reserves kCountLds
// bytes of LDS that the kernel never touches, so that at most three
// workgroups are resident per CU: with nothing else to do, fewer
// workgroups in flight read faster (on 8.19 G words 4.49 ms at three per
// CU, 4.56-4.63 ms at four, 4.68 ms at eight, 5.2 ms at two).
constexpr size_t kCountLds = 48 * 1024;
template <bool kMulti, bool kVec>
__global__ __launch_bounds__(kThreads) void count_kernel(ExtractArgs a) {
  __shared__ uint32_t s_wave_total[kWaves];
  const uint64_t tile = xcd_tile(blockIdx.x, a.num_tiles);
  const TensorDesc d = tile_desc<kMulti>(a, tile);
  TileScan s;
  scan_tile<kVec>(d, tile, lane_id(), threadIdx.x >> 6, s_wave_total, s);
  if (threadIdx.x == 0) a.counts[tile] = s.tile_total;
}

// ----------------------------------------------------------------- scan

// Sum of the counts of each group of kTilesPerGroup tiles (one wavefront).
template <typename CountT>
__global__ __launch_bounds__(64) void group_sum_kernel(const CountT* counts, uint64_t num_tiles,
                                                       uint64_t* group_sum) {
  const uint64_t t = (uint64_t)blockIdx.x * kTilesPerGroup + threadIdx.x;
  const uint64_t c = t < num_tiles ? (uint64_t)counts[t] : 0;
  const uint64_t s = wave_sum64(c);
  if (threadIdx.x == 0) group_sum[blockIdx.x] = s;
}

// Exclusive scan of the group sums by one workgroup, also writing the
// total.  Wavefront w owns a contiguous range of the sums, in blocks of 64
// (one per lane, loaded coalesced, kScanBatch blocks in flight at a time).
// Pass 1: each wavefront sums its range; the range sums are combined
// through LDS.  Pass 2: each wavefront scans its blocks in order, carrying
// the running offset, and writes the exclusive offsets.
constexpr int kScanThreads = 1024;
constexpr int kScanWaves = kScanThreads / 64;
constexpr int kScanBatch = 8;
__global__ __launch_bounds__(kScanThreads) void group_scan_kernel(const uint64_t* group_sum,
                                                                  uint64_t num_groups,
                                                                  uint64_t* group_excl,
                                                                  uint64_t* d_count) {
  __shared__ uint64_t s_wave[kScanWaves];
  const uint32_t lane = lane_id();
  const uint32_t wave = threadIdx.x >> 6;
  const uint64_t blocks = (num_groups + 63) / 64;
  const uint64_t per = (blocks + kScanWaves - 1) / kScanWaves;   // blocks per wavefront
  const uint64_t b0 = (uint64_t)wave * per;
  const uint64_t b1 = b0 + per < blocks ? b0 + per : blocks;
  uint64_t part = 0;
  for (uint64_t b = b0; b < b1; b += kScanBatch) {
    uint64_t v[kScanBatch];
#pragma unroll
    for (int k = 0; k < kScanBatch; ++k) {
      const uint64_t i = (b + k) * 64 + lane;
      v[k] = (b + k < b1 && i < num_groups) ? group_sum[i] : 0;
    }
#pragma unroll
    for (int k = 0; k < kScanBatch; ++k) part += v[k];
  }
  part = wave_sum64(part);
  if (lane == 0) s_wave[wave] = part;
  __syncthreads();
  uint64_t carry = 0, total = 0;
  for (uint32_t w = 0; w < (uint32_t)kScanWaves; ++w) {
    const uint64_t t = s_wave[w];
    carry += w < wave ? t : 0;
    total += t;
  }
  for (uint64_t b = b0; b < b1; b += kScanBatch) {
    uint64_t v[kScanBatch];
#pragma unroll
    for (int k = 0; k < kScanBatch; ++k) {
      const uint64_t i = (b + k) * 64 + lane;
      v[k] = (b + k < b1 && i < num_groups) ? group_sum[i] : 0;
    }
#pragma unroll
    for (int k = 0; k < kScanBatch; ++k) {
      uint64_t x = v[k];   // inclusive scan of the block within the wavefront
#pragma unroll
      for (int s = 1; s < 64; s <<= 1) {
        const uint64_t y = __shfl_up(x, s);
        if ((int)lane >= s) x += y;
      }
      const uint64_t i = (b + k) * 64 + lane;
      if (b + k < b1 && i < num_groups) group_excl[i] = carry + x - v[k];
      carry += __shfl(x, 63);
    }
  }
  if (threadIdx.x == 0) *d_count = total;
}

// Up to 1024 groups (65536 tiles): the group sums and their scan in one
// workgroup, one launch instead of two.  Wavefront w sums groups w, w + 16,
// ... (4 of them per round, loads coalesced), into LDS; then every thread
// scans one group.
constexpr uint64_t kSmallScanGroups = kScanThreads;

template <typename CountT>
__global__ __launch_bounds__(kScanThreads) void tile_scan_kernel(const CountT* counts,
                                                                 uint64_t num_tiles,
                                                                 uint64_t* group_excl,
                                                                 uint64_t* d_count) {
  __shared__ uint64_t s_g[kSmallScanGroups];
  __shared__ uint64_t s_wave[kScanWaves];
  const uint32_t lane = lane_id();
  const uint32_t wave = threadIdx.x >> 6;
  const uint64_t groups = groups_for(num_tiles);
  for (uint64_t g0 = wave; g0 < groups; g0 += 4 * kScanWaves) {
    uint64_t v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint64_t g = g0 + k * kScanWaves;
      const uint64_t t = g * kTilesPerGroup + lane;
      v[k] = (g < groups && t < num_tiles) ? (uint64_t)counts[t] : 0;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint64_t g = g0 + k * kScanWaves;
      const uint64_t sum = wave_sum64(v[k]);
      if (lane == 0 && g < groups) s_g[g] = sum;
    }
  }
  __syncthreads();
  const uint64_t x0 = threadIdx.x < groups ? s_g[threadIdx.x] : 0;
  uint64_t x = x0;
#pragma unroll
  for (int s = 1; s < 64; s <<= 1) {
    const uint64_t y = __shfl_up(x, s);
    if ((int)lane >= s) x += y;
  }
  if (lane == 63) s_wave[wave] = x;
  __syncthreads();
  uint64_t carry = 0;
  for (uint32_t w = 0; w < wave; ++w) carry += s_wave[w];
  if (threadIdx.x < groups) group_excl[threadIdx.x] = carry + x - x0;
  if (threadIdx.x == kScanThreads - 1) *d_count = carry + x;
}

// ------------------------------------------------------------- finalize

// Output index of word 0 of `tile`, read by one lane (tile ids differ per
// lane here, so the descriptor stays in vector registers).
template <bool kMulti>
__device__ __forceinline__ TensorDesc lane_desc(const ExtractArgs& a, uint64_t tile) {
  return kMulti ? a.table[a.tile_map[tile]] : a.inl[inline_row(a, tile)];
}

constexpr int kFinBatch = 8;

// Calls over at most kOwnScanGroups groups (2^28 words: the pipeline's
// chunks) launch no scan between the stage and finalize kernels: each
// finalize workgroup sums the tile counts before its own group itself (at
// most 128 KiB, just written by the stage kernel), and the last group's
// workgroup writes the total.  A one-workgroup scan is a chain of
// dependent loads plus a launch; beside a running stage kernel (the
// pipeline's next chunk) it took 50-90 us per chunk.
constexpr uint64_t kOwnScanGroups = 512;

// Sum of counts[0, t0) over the workgroup (every thread gets it); t0 is a
// multiple of kTilesPerGroup and counts 16-byte aligned, so the range is
// whole 16-byte vectors, loaded eight per thread at a time.
constexpr int kOwnScanBatch = 8;
__device__ __forceinline__ uint64_t counts_before_group(const uint32_t* counts, uint64_t t0,
                                                        uint64_t* s_part) {
  const u32x4* c4 = reinterpret_cast<const u32x4*>(counts);
  const uint64_t n4 = t0 / 4;
  uint64_t v = 0;
  for (uint64_t i0 = threadIdx.x; i0 < n4; i0 += (uint64_t)kThreads * kOwnScanBatch) {
    u32x4 w[kOwnScanBatch];
#pragma unroll
    for (int k = 0; k < kOwnScanBatch; ++k) {
      const uint64_t i = i0 + (uint64_t)kThreads * k;
      w[k] = i < n4 ? c4[i] : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int k = 0; k < kOwnScanBatch; ++k)
      v += (uint64_t)w[k][0] + (uint64_t)w[k][1] + (uint64_t)w[k][2] + (uint64_t)w[k][3];
  }
  v = wave_sum64(v);
  if (lane_id() == 0) s_part[threadIdx.x >> 6] = v;
  __syncthreads();
  uint64_t total = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) total += s_part[w];
  return total;
}

template <typename IdxT, bool kMulti, bool kVec, bool kOwnScan>
__global__ __launch_bounds__(kThreads) void finalize_kernel(ExtractArgs a) {
  __shared__ uint32_t s_begin[kTilesPerGroup + 1];   // run start of each tile in the group
  __shared__ uint32_t s_count[kTilesPerGroup];
  __shared__ int64_t s_out_base[kTilesPerGroup];
  __shared__ uint32_t s_wave_total[kWaves];
  __shared__ uint64_t s_part[kWaves];
  const uint64_t groups = (a.num_tiles + kTilesPerGroup - 1) / kTilesPerGroup;
  const uint64_t g = xcd_tile(blockIdx.x, groups);
  const uint64_t t0 = g * kTilesPerGroup;
  const uint64_t left = a.num_tiles - t0;
  const uint32_t n_here = left < (uint64_t)kTilesPerGroup ? (uint32_t)left : kTilesPerGroup;
  const uint32_t lane = lane_id();
  const uint32_t wave = threadIdx.x >> 6;
  const uint64_t group_excl = kOwnScan ? counts_before_group(a.counts, t0, s_part)
                                       : a.group_excl[g];
  if (wave == 0) {
    // exclusive scan of the group's tile counts (one tile per lane)
    const uint64_t t = t0 + lane;
    const bool in = lane < n_here;
    const uint32_t c = in ? a.counts[t] : 0u;
    uint32_t x = c;
#pragma unroll
    for (int s = 1; s < 64; s <<= 1) {
      const uint32_t y = __shfl_up(x, s);
      if ((int)lane >= s) x += y;
    }
    s_begin[lane] = x - c;
    if (lane == 63) s_begin[64] = x;
    s_count[lane] = c;
    if (in) {
      const TensorDesc d = lane_desc<kMulti>(a, t);
      s_out_base[lane] = tile_out_base(d, t);
      if (a.d_tensor_offsets) {
        // tensor_offsets: the first tile of a slice owns the slots of its
        // own tensor and of the empty tensors just before it; the last tile
        // owns the slots after its tensor (trailing empty tensors, total).
        const uint64_t excl = group_excl + (x - c);
        if (t == d.first_tile)
          for (uint32_t s = d.off_lo; s <= d.slot; ++s) a.d_tensor_offsets[s] = excl;
        if (t == a.num_tiles - 1)
          for (uint32_t s = d.slot + 1; s <= a.num_tensors; ++s) a.d_tensor_offsets[s] = excl + c;
      }
    }
  }
  __syncthreads();
  IdxT* out_idx = reinterpret_cast<IdxT*>(a.out_idx);
  const uint32_t total = s_begin[64];
  if (kOwnScan && g == groups - 1 && threadIdx.x == 0) *a.d_count = group_excl + total;
  // Every staged entry of the group, in output order, spread over all
  // threads; the tile of entry e is found by binary search over s_begin.
  // Each thread loads kFinBatch entries before it stores any, so that many
  // loads are in flight.  Entries of overflowed tiles are skipped here and
  // written below.
  for (uint32_t e0 = 0; e0 < total; e0 += kThreads * kFinBatch) {
    uint32_t v[kFinBatch], ti[kFinBatch];
#pragma unroll
    for (int k = 0; k < kFinBatch; ++k) {
      const uint32_t e = e0 + threadIdx.x + kThreads * k;
      uint32_t lo = 0, hi = 64;   // s_begin[lo] <= e < s_begin[hi]
#pragma unroll
      for (int step = 0; step < 6; ++step) {
        const uint32_t mid = (lo + hi) >> 1;
        if (s_begin[mid] <= e) lo = mid; else hi = mid;
      }
      ti[k] = lo;
      const bool take = e < total && s_count[lo] <= a.stage_cap && group_excl + e < a.capacity;
      v[k] = take ? __builtin_nontemporal_load(a.stage + (t0 + lo) * a.stage_stride +
                                               (e - s_begin[lo]))
                  : 0u;
    }
#pragma unroll
    for (int k = 0; k < kFinBatch; ++k) {
      const uint32_t e = e0 + threadIdx.x + kThreads * k;
      const uint32_t i = ti[k];
      if (e < total && s_count[i] <= a.stage_cap && group_excl + e < a.capacity) {
        out_idx[group_excl + e] = (IdxT)(s_out_base[i] + (v[k] & 0xFFFFu));
        a.out_val[group_excl + e] = (uint16_t)(v[k] >> 16);
      }
    }
  }
  // Tiles that overflowed their slot: read again and write every entry.
  for (uint32_t i = 0; i < n_here; ++i) {
    if (s_count[i] <= a.stage_cap) continue;
    const uint64_t tile = t0 + i;
    const TensorDesc d = tile_desc<kMulti>(a, tile);
    TileScan s;
    scan_tile<kVec>(d, tile, lane, wave, s_wave_total, s);
    const int64_t lane_out = s_out_base[i] + (int64_t)(wave * kGroupsPerWave + lane) * 8;
    const uint64_t excl = group_excl + s_begin[i];
#pragma unroll
    for (int u = 0; u < kChunks; ++u) {
      uint32_t m = s.mask[u];
      uint64_t pos = excl + s.rank[u];
      const int64_t e0 = lane_out + 512 * u;
      while (m) {
        const int j = __builtin_ctz(m);
        m &= m - 1;
        if (pos < a.capacity) {
          out_idx[pos] = (IdxT)(e0 + j);
          a.out_val[pos] = word_of(s.q[u], j);
        }
        ++pos;
      }
    }
    __syncthreads();   // s_wave_total is reused by the next overflowed tile
  }
}

// -------------------------------------------------- small single-tensor calls
//
// A call over few tiles is bound by its launches, not by memory: the
// group scan and a finalize of one workgroup per 64 tiles (8 workgroups
// for a 2048 x 2048 tensor) cost more than the scan itself.  For one
// tensor over at most kSmallTiles tiles, finalize_small runs one workgroup
// per tile after the stage kernel: it sums the counts of the tiles before
// its own (read from L2) and copies its slot, two launches in all.

// Sum of counts[0, n) over the workgroup (every thread gets it).
__device__ __forceinline__ uint64_t sum_counts_before(const uint32_t* counts, uint64_t n,
                                                      uint64_t* s_part) {
  uint64_t v = 0;
  for (uint64_t i = threadIdx.x; i < n; i += kThreads) v += counts[i];
  v = wave_sum64(v);
  if (lane_id() == 0) s_part[threadIdx.x >> 6] = v;
  __syncthreads();
  uint64_t total = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) total += s_part[w];
  return total;
}

// Writes one tile's entries in output order straight from a tile scan,
// entry r of the tile at position excl + r (for a tile that overflowed its
// staging slot).
template <typename IdxT>
__device__ __forceinline__ void write_scanned_tile(const ExtractArgs& a, const TileScan& s,
                                                   int64_t lane_out, uint64_t excl) {
  IdxT* out_idx = reinterpret_cast<IdxT*>(a.out_idx);
#pragma unroll
  for (int u = 0; u < kChunks; ++u) {
    uint32_t m = s.mask[u];
    uint64_t pos = excl + s.rank[u];
    const int64_t e0 = lane_out + 512 * u;
    while (m) {
      const int j = __builtin_ctz(m);
      m &= m - 1;
      if (pos < a.capacity) {
        out_idx[pos] = (IdxT)(e0 + j);
        a.out_val[pos] = word_of(s.q[u], j);
      }
      ++pos;
    }
  }
}

template <typename IdxT, bool kVec>
__global__ __launch_bounds__(kThreads) void finalize_small_kernel(ExtractArgs a) {
  __shared__ uint64_t s_part[kWaves];
  __shared__ uint32_t s_wave_total[kWaves];
  const uint64_t tile = blockIdx.x;
  const uint64_t excl = sum_counts_before(a.counts, tile, s_part);
  const uint32_t count = a.counts[tile];
  if (tile == a.num_tiles - 1 && threadIdx.x == 0) *a.d_count = excl + count;
  const TensorDesc d = a.inl[0];
  const int64_t base = tile_out_base(d, tile);
  IdxT* out_idx = reinterpret_cast<IdxT*>(a.out_idx);
  if (count <= a.stage_cap) {
    const uint32_t* slot = a.stage + tile * a.stage_stride;
    for (uint32_t r = threadIdx.x; r < count; r += kThreads) {
      if (excl + r >= a.capacity) break;
      const uint32_t v = __builtin_nontemporal_load(slot + r);
      out_idx[excl + r] = (IdxT)(base + (v & 0xFFFFu));
      a.out_val[excl + r] = (uint16_t)(v >> 16);
    }
  } else {
    // the tile overflowed its slot: read it again
    const uint32_t lane = lane_id(), wave = threadIdx.x >> 6;
    TileScan s;
    scan_tile<kVec>(d, tile, lane, wave, s_wave_total, s);
    write_scanned_tile<IdxT>(a, s, base + (int64_t)(wave * kGroupsPerWave + lane) * 8, excl);
  }
}

// ------------------------------------------------------------ coded output
//
// The chunked pipeline's coded form (gap + LEB128, one segment per call,
// Sec. 5.1 "Sparse encoding") written straight from the staging slots: no
// index stream is formed.  An entry's code is that of its gap: the index
// minus the previous kept index, or minus code_base for the first entry.
// Inside a tile the gaps come from the staged offsets; a tile's first entry
// is coded against the last kept index of the nearest earlier tile that
// kept anything, found by a running maximum of the tiles' last indices
// (indices grow with the tile id; code_base starts the maximum, as every
// index is at least code_base).

__device__ __forceinline__ uint32_t leb_bytes(uint64_t v) {
  const uint32_t bits = 64 - __builtin_clzll(v | 1ull);
  return (bits + 6) / 7;
}

// Last kept index of the nearest lower lane that kept anything (-1: none)
// and of the highest such lane, where `last` is -1 for lanes that kept
// nothing.  Kept indices grow with the lane, so these are the exclusive and
// the total maximum of `last` over the wavefront: one ballot and one
// shuffle instead of a scan.
__device__ __forceinline__ void lower_last(int64_t last, uint32_t lane, int64_t& before,
                                           int64_t& top) {
  const uint64_t nz = __ballot(last >= 0);
  const uint64_t below = nz & ((1ull << lane) - 1ull);
  const int src = below ? 63 - __builtin_clzll(below) : (int)lane;
  const int64_t b = __shfl(last, src);
  before = below ? b : -1;
  top = nz ? __shfl(last, 63 - __builtin_clzll(nz)) : -1;
}

template <typename T>
__device__ __forceinline__ T wave_incl_sum(T x, uint32_t lane) {
#pragma unroll
  for (int s = 1; s < 64; s <<= 1) {
    const T y = __shfl_up(x, s);
    if ((int)lane >= s) x += y;
  }
  return x;
}

// Index a tile's first entry is coded against, given the last kept index
// before it (-1: none): with one segment per tensor, never below the
// tensor's word 0, so that a tensor's first entry is coded as its
// tensor-local index.
__device__ __forceinline__ int64_t coded_pred(const ExtractArgs& a, int64_t before,
                                              int64_t seg_base) {
  return (a.seg_per_tensor && seg_base > before) ? seg_base : before;
}

// Descriptor of `tile`'s slice (tile ids differ per lane).
__device__ __forceinline__ TensorDesc any_desc(const ExtractArgs& a, uint64_t tile) {
  return a.table ? a.table[a.tile_map[tile]] : a.inl[inline_row(a, tile)];
}

// Per group of kTilesPerGroup tiles (one wavefront each): its entries, the
// code bytes of every entry whose predecessor lies in the group, its last
// (largest) index and the first index of its first tile that kept
// anything; that first entry's code length is settled by the scan, once
// the group's predecessor index is known (with one segment per tensor, the
// group's first entry is never coded against less than its tensor-local
// index, kept in group_first_local).  Written into the tables the scan
// then overwrites in place: group_sum = entries | bytes << 32, group_prev =
// last index, group_bexcl = first index (-1: none kept).
__global__ __launch_bounds__(64) void coded_group_kernel(ExtractArgs a) {
  const uint32_t lane = lane_id();
  const uint64_t g = blockIdx.x;
  const uint64_t t = g * kTilesPerGroup + lane;
  const bool in = t < a.num_tiles;
  const uint64_t rec = in ? a.tile_rec[t] : 0;
  const uint32_t c = rec_count(rec);
  int64_t f = 0, l = 0, seg_base = -1;
  if (c) {
    const TensorDesc d = any_desc(a, t);
    const int64_t ob = tile_out_base(d, t);
    f = ob + (int64_t)rec_first(rec);
    l = ob + (int64_t)rec_last(rec);
    if (a.seg_per_tensor) seg_base = (int64_t)d.seg_base;
  }
  int64_t before, last;
  lower_last(c ? l : -1, lane, before, last);
  const uint64_t inner = rec_inner(rec);
  const uint64_t own =
      c ? inner + (before >= 0 ? leb_bytes((uint64_t)(f - coded_pred(a, before, seg_base))) : 0u)
        : 0u;
  const uint64_t nz = __ballot(c != 0);
  const int first_lane = nz ? (int)__builtin_ctzll(nz) : 0;
  const int64_t first = nz ? __shfl(f, first_lane) : -1;
  const int64_t first_local = nz ? __shfl(f - seg_base, first_lane) : 0;
  const uint64_t cnt = wave_sum64(c);
  const uint64_t bytes = wave_sum64(own);
  if (lane == 0) {
    a.group_sum[g] = cnt | (bytes << 32);
    a.group_prev[g] = last;
    a.group_bexcl[g] = (uint64_t)first;
    if (a.seg_per_tensor) a.group_first_local[g] = first_local;
  }
}

// Code length of a group's (or tile's) first entry, given the index it
// follows: the gap from it, or (one segment per tensor) the tensor-local
// index if that is smaller.
__device__ __forceinline__ uint32_t first_entry_bytes(const ExtractArgs& a, int64_t first,
                                                      int64_t prev, int64_t local) {
  int64_t gap = first - prev;
  if (a.seg_per_tensor && local < gap) gap = local;
  return leb_bytes((uint64_t)gap);
}

// One block of 64 groups of the coded scan, one per lane.
struct CodedBlock {
  uint64_t packed;   // entries | code bytes of every entry but the first << 32
  int64_t last;      // last kept index (-1: none)
  int64_t first;     // first kept index (-1: none)
  int64_t local;     // its tensor-local index (one segment per tensor)
};

__device__ __forceinline__ CodedBlock load_coded_block(const ExtractArgs& a, uint64_t gi,
                                                       bool in) {
  CodedBlock b;
  b.packed = in ? a.group_sum[gi] : 0;
  b.last = in ? a.group_prev[gi] : -1;
  b.first = in ? (int64_t)a.group_bexcl[gi] : -1;
  b.local = (in && a.seg_per_tensor) ? a.group_first_local[gi] : 0;
  return b;
}

// One workgroup of kScanWaves wavefronts: per group, the entries and code
// bytes before it and the index its first entry is coded against (the
// largest kept index of the groups before it, at least code_base); the
// totals.  Wavefront w owns a contiguous range of groups, in blocks of 64
// (one per lane, kScanBatch blocks loaded at a time).  Inside a range, a
// group's predecessor index lies in the range once any earlier group of
// the range kept something, so only the range's first nonempty group
// depends on the ranges before it.  Pass 1: each wavefront sums its
// range's entries and code bytes, leaving out that one group's first
// entry, and takes the range's largest index.  The ranges are then
// chained (sixteen steps, in every thread), which settles each range's
// deferred entry.  Pass 2: each wavefront walks its range again with its
// carries and writes every group's offsets (a thread reads its group's
// sums before it overwrites them, and pass 1 has read everything before
// the barrier).
__global__ __launch_bounds__(kScanThreads) void coded_scan_kernel(ExtractArgs a) {
  __shared__ uint64_t s_cnt[kScanWaves], s_bytes[kScanWaves];
  __shared__ int64_t s_max[kScanWaves], s_dfirst[kScanWaves], s_dlocal[kScanWaves];
  const uint32_t lane = lane_id();
  const uint32_t wave = threadIdx.x >> 6;
  const uint64_t groups = groups_for(a.num_tiles);
  const uint64_t blocks = (groups + 63) / 64;
  const uint64_t per = (blocks + kScanWaves - 1) / kScanWaves;   // blocks per wavefront
  const uint64_t b0 = (uint64_t)wave * per;
  const uint64_t b1 = b0 + per < blocks ? b0 + per : blocks;
  // pass 1
  uint64_t cnt = 0, bytes = 0;
  int64_t run_max = -1, dfirst = -1, dlocal = 0;
  for (uint64_t b = b0; b < b1; b += kScanBatch) {
    CodedBlock v[kScanBatch];
#pragma unroll
    for (int k = 0; k < kScanBatch; ++k) {
      const uint64_t gi = (b + k) * 64 + lane;
      v[k] = load_coded_block(a, gi, b + k < b1 && gi < groups);
    }
#pragma unroll
    for (int k = 0; k < kScanBatch; ++k) {
      int64_t before, bmax;
      lower_last(v[k].last, lane, before, bmax);
      const int64_t pred = before > run_max ? before : run_max;
      uint64_t own = v[k].packed >> 32;
      if (v[k].first >= 0 && pred >= 0) own += first_entry_bytes(a, v[k].first, pred, v[k].local);
      // the range's first nonempty group: at most one lane of one block
      const uint64_t defer = __ballot(v[k].first >= 0 && pred < 0);
      if (defer) {
        const int l = (int)__builtin_ctzll(defer);
        dfirst = __shfl(v[k].first, l);
        dlocal = __shfl(v[k].local, l);
      }
      cnt += v[k].packed & 0xFFFFFFFFull;
      bytes += own;
      run_max = bmax > run_max ? bmax : run_max;
    }
  }
  cnt = wave_sum64(cnt);
  bytes = wave_sum64(bytes);
  if (lane == 0) {
    s_cnt[wave] = cnt;
    s_bytes[wave] = bytes;
    s_max[wave] = run_max;
    s_dfirst[wave] = dfirst;
    s_dlocal[wave] = dlocal;
  }
  __syncthreads();
  // chain the ranges
  uint64_t carry_cnt = 0, carry_bytes = 0, total_cnt = 0, total_bytes = 0;
  int64_t carry_prev = a.code_base, prev = a.code_base;
  for (uint32_t w = 0; w < (uint32_t)kScanWaves; ++w) {
    if (w == wave) {
      carry_cnt = total_cnt;
      carry_bytes = total_bytes;
      carry_prev = prev;
    }
    uint64_t rb = s_bytes[w];
    if (s_dfirst[w] >= 0) rb += first_entry_bytes(a, s_dfirst[w], prev, s_dlocal[w]);
    total_cnt += s_cnt[w];
    total_bytes += rb;
    prev = s_max[w] > prev ? s_max[w] : prev;
  }
  // pass 2
  for (uint64_t b = b0; b < b1; b += kScanBatch) {
    CodedBlock v[kScanBatch];
#pragma unroll
    for (int k = 0; k < kScanBatch; ++k) {
      const uint64_t gi = (b + k) * 64 + lane;
      v[k] = load_coded_block(a, gi, b + k < b1 && gi < groups);
    }
#pragma unroll
    for (int k = 0; k < kScanBatch; ++k) {
      int64_t before, bmax;
      lower_last(v[k].last, lane, before, bmax);
      const int64_t pred = before > carry_prev ? before : carry_prev;
      // a group holds at most 2^19 entries of at most 2 code bytes each
      // (plus one longer number), so a block's sums fit 32 bits
      const uint32_t c = (uint32_t)(v[k].packed & 0xFFFFFFFFull);
      const uint32_t own = (uint32_t)(v[k].packed >> 32) +
                           (v[k].first >= 0 ? first_entry_bytes(a, v[k].first, pred, v[k].local)
                                            : 0u);
      const uint32_t xc = wave_incl_sum(c, lane);
      const uint32_t xb = wave_incl_sum(own, lane);
      const uint64_t gi = (b + k) * 64 + lane;
      if (b + k < b1 && gi < groups) {
        a.group_excl[gi] = carry_cnt + xc - c;
        a.group_bexcl[gi] = carry_bytes + xb - own;
        a.group_prev[gi] = pred;
      }
      carry_cnt += __shfl(xc, 63);
      carry_bytes += __shfl(xb, 63);
      carry_prev = bmax > carry_prev ? bmax : carry_prev;
    }
  }
  if (threadIdx.x == 0) {
    *a.d_count = total_cnt;
    *a.d_nbytes = total_bytes;
  }
}

// A group's entries are coded in windows of kCodeWin consecutive entries,
// kCodePer per thread.  A window's code is at most two bytes per entry plus
// the longer codes of at most one first entry per tile (an index gap of
// up to 2^63 takes 9 bytes).
constexpr int kCodePer = 8;
constexpr int kCodeWin = kThreads * kCodePer;
constexpr int kCodeWinBytes = 2 * kCodeWin + kTilesPerGroup * 8;

// Window entry j sits at win[wslot(j)]: one padding word after every
// kCodePer entries, so that the threads of a wavefront, each walking its
// own kCodePer consecutive entries, read different LDS banks.
constexpr uint32_t kWinPad = 1;
__device__ __forceinline__ uint32_t wslot(uint32_t j) { return kWinPad ? j + j / kCodePer : j; }

struct CodedGroup {
  uint32_t begin[kTilesPerGroup + 1];   // first entry of each tile within the group, total
  uint32_t count[kTilesPerGroup];
  int64_t out_base[kTilesPerGroup];     // index of word 0 of each tile
  int64_t prev[kTilesPerGroup];         // index each tile's first entry is coded against
  uint32_t win[kCodeWin + kCodeWin / kCodePer];   // the window's entries, (word << 16) | offset
  uint8_t code[kCodeWinBytes];
  uint32_t wave_total[kWaves];
  uint32_t last_off;                    // offset of the previous window's last entry
  uint32_t overflow;
  uint64_t eg, bg;                      // entries and code bytes before the group (own scan)
};

// The coded scan for one group, by one wavefront of its finalize workgroup
// (calls over at most kOwnScanGroups groups): the entries and code bytes
// of groups [0, g) and the index group g's first entry is coded against,
// from the records coded_group_kernel left, walked in blocks of 64 groups
// as the second pass of coded_scan_kernel walks them.
constexpr int kOwnCodedBatch = 4;
__device__ __forceinline__ void own_coded_scan(const ExtractArgs& a, uint64_t g, uint32_t lane,
                                               uint64_t& eg, uint64_t& bg, int64_t& gp) {
  uint64_t cnt = 0, bytes = 0;
  int64_t carry_prev = a.code_base;
  for (uint64_t b = 0; b * 64 < g; b += kOwnCodedBatch) {
    CodedBlock v[kOwnCodedBatch];
#pragma unroll
    for (int k = 0; k < kOwnCodedBatch; ++k) {
      const uint64_t gi = (b + k) * 64 + lane;
      v[k] = load_coded_block(a, gi, gi < g);
    }
#pragma unroll
    for (int k = 0; k < kOwnCodedBatch; ++k) {
      int64_t before, bmax;
      lower_last(v[k].last, lane, before, bmax);
      const int64_t pred = before > carry_prev ? before : carry_prev;
      cnt += v[k].packed & 0xFFFFFFFFull;
      bytes += (v[k].packed >> 32) +
               (v[k].first >= 0 ? first_entry_bytes(a, v[k].first, pred, v[k].local) : 0u);
      carry_prev = bmax > carry_prev ? bmax : carry_prev;
    }
  }
  eg = wave_sum64(cnt);
  bg = wave_sum64(bytes);
  gp = carry_prev;
}

// Stores bytes [0, n) of `src` at dst (4-byte stores where dst is aligned).
__device__ __forceinline__ void flush_code(const uint8_t* src, uint32_t n, uint8_t* dst) {
  const uint32_t head = (uint32_t)((4u - ((uintptr_t)dst & 3u)) & 3u);
  const uint32_t h = head < n ? head : n;
  const uint32_t words = (n - h) / 4;
  for (uint32_t i = threadIdx.x; i < h; i += kThreads) dst[i] = src[i];
  uint32_t* dw = reinterpret_cast<uint32_t*>(dst + h);
  for (uint32_t w = threadIdx.x; w < words; w += kThreads) {
    const uint32_t j = h + 4 * w;
    dw[w] = (uint32_t)src[j] | ((uint32_t)src[j + 1] << 8) | ((uint32_t)src[j + 2] << 16) |
            ((uint32_t)src[j + 3] << 24);
  }
  for (uint32_t i = h + 4 * words + threadIdx.x; i < n; i += kThreads) dst[i] = src[i];
}

// Walks the kCodePer consecutive window entries of this thread, from
// window entry j0 on, calling f(k, gap) for each entry inside the window:
// a tile's first entry is coded against the tile's predecessor index, any
// other entry against the entry before it.
template <typename F>
__device__ __forceinline__ void walk_gaps(const CodedGroup& sg, uint32_t e_lo, uint32_t n,
                                          uint32_t j0, F f) {
  uint32_t lo = 0, hi = kTilesPerGroup;   // begin[lo] <= e_lo + j0 < begin[hi]
#pragma unroll
  for (int step = 0; step < 6; ++step) {
    const uint32_t mid = (lo + hi) >> 1;
    if (sg.begin[mid] <= e_lo + j0) lo = mid; else hi = mid;
  }
  uint32_t ti = lo;
  uint32_t prev_off = j0 > 0 ? (sg.win[wslot(j0 - 1)] & 0xFFFFu) : sg.last_off;
#pragma unroll
  for (int k = 0; k < kCodePer; ++k) {
    const uint32_t j = j0 + k;
    if (j < n) {
      const uint32_t e = e_lo + j;
      while (e >= sg.begin[ti + 1]) ++ti;
      const uint32_t off = sg.win[wslot(j)] & 0xFFFFu;
      f(k, e == sg.begin[ti] ? (uint64_t)(sg.out_base[ti] + (int64_t)off - sg.prev[ti])
                             : (uint64_t)(off - prev_off));
      prev_off = off;
    }
  }
}

// Codes the window of n entries that starts at group entry e_lo (entries in
// sg.win): values to out_val, code bytes after the `written` bytes the
// group has already put out.  Returns the window's code bytes.  The gaps
// are walked twice (lengths, then bytes) rather than held in registers.
__device__ __forceinline__ uint32_t code_window(const ExtractArgs& a, CodedGroup& sg,
                                                uint32_t e_lo, uint32_t n, uint64_t eg,
                                                uint64_t bg, uint64_t written) {
  const uint32_t lane = lane_id();
  const uint32_t wave = threadIdx.x >> 6;
  const uint32_t j0 = kCodePer * threadIdx.x;
  uint32_t sum = 0;
  if (j0 < n) walk_gaps(sg, e_lo, n, j0, [&](int, uint64_t gap) { sum += leb_bytes(gap); });
  // the window's words, one entry per thread in turn (coalesced stores)
  for (uint32_t j = threadIdx.x; j < n; j += kThreads)
    if (eg + e_lo + j < a.capacity) a.out_val[eg + e_lo + j] = (uint16_t)(sg.win[wslot(j)] >> 16);
  const uint32_t incl = wave_incl_sum(sum, lane);
  if (lane == 63) sg.wave_total[wave] = incl;
  __syncthreads();
  uint32_t pos = incl - sum, nb = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    pos += (uint32_t)w < wave ? sg.wave_total[w] : 0u;
    nb += sg.wave_total[w];
  }
  if (j0 < n) {
    walk_gaps(sg, e_lo, n, j0, [&](int, uint64_t gap) {
      const uint32_t len = leb_bytes(gap);
      for (uint32_t m = 0; m < len; ++m) {
        sg.code[pos++] = (uint8_t)((gap & 0x7Fu) | (m + 1 < len ? 0x80u : 0u));
        gap >>= 7;
      }
    });
  }
  __syncthreads();
  const uint64_t at = bg + written;
  const uint64_t room = a.code_capacity > at ? a.code_capacity - at : 0;
  flush_code(sg.code, room < nb ? (uint32_t)room : nb, a.code_out + at);
  if (threadIdx.x == 0) sg.last_off = sg.win[wslot(n - 1)] & 0xFFFFu;
  __syncthreads();
  return nb;
}

// One workgroup per group: the window entries come from the staging slots,
// loaded kCodePer per thread at a time.  A group with a tile that
// overflowed its slot is coded tile by tile instead, that tile read again
// and its entries placed into the window by rank.  The launch bound asks
// for six wavefronts per SIMD (at most 80 registers): measured faster than
// the five the unbounded allocation gives.
template <bool kMulti, bool kVec, bool kOwnScan>
__global__ __launch_bounds__(kThreads, 6) void finalize_coded_kernel(ExtractArgs a) {
  __shared__ CodedGroup sg;
  __shared__ uint32_t s_wave_total[kWaves];
  const uint64_t groups = (a.num_tiles + kTilesPerGroup - 1) / kTilesPerGroup;
  const uint64_t g = blockIdx.x;
  const uint64_t t0 = g * kTilesPerGroup;
  const uint64_t left = a.num_tiles - t0;
  const uint32_t n_here = left < (uint64_t)kTilesPerGroup ? (uint32_t)left : kTilesPerGroup;
  const uint32_t lane = lane_id();
  const uint32_t wave = threadIdx.x >> 6;
  uint64_t eg = 0, bg = 0;
  if (!kOwnScan) {
    eg = a.group_excl[g];
    bg = a.group_bexcl[g];
  }
  if (wave == 0) {
    int64_t gp;
    if (kOwnScan) {
      own_coded_scan(a, g, lane, eg, bg, gp);
      if (lane == 0) {
        sg.eg = eg;
        sg.bg = bg;
      }
    } else {
      gp = a.group_prev[g];
    }
    const uint64_t t = t0 + lane;
    const bool in = lane < n_here;
    const uint64_t rec = in ? a.tile_rec[t] : 0;
    const uint32_t c = rec_count(rec);
    TensorDesc d = {};
    int64_t ob = 0;
    if (in) {
      d = lane_desc<kMulti>(a, t);
      ob = tile_out_base(d, t);
    }
    int64_t before, top;
    lower_last(c ? ob + (int64_t)rec_last(rec) : -1, lane, before, top);
    if (before < gp) before = gp;
    const uint32_t x = wave_incl_sum(c, lane);
    const int64_t prev = in ? coded_pred(a, before, (int64_t)d.seg_base) : before;
    sg.begin[lane] = x - c;
    if (lane == 63) sg.begin[64] = x;
    sg.count[lane] = c;
    sg.prev[lane] = prev;
    sg.out_base[lane] = ob;
    const uint64_t over = __ballot(c > a.stage_cap);
    if (lane == 0) {
      sg.overflow = over != 0;
      sg.last_off = 0;
    }
    if (a.seg_per_tensor && (a.d_tensor_offsets || a.d_tensor_byte_offsets)) {
      // Entry and byte offsets of each tensor's segment: the first tile of
      // a slice owns the slots of its tensor and of the empty tensors just
      // before it; the last tile owns the slots after its tensor.  A tile's
      // code is its inner gaps plus its first entry's number.
      const int64_t f = ob + (int64_t)rec_first(rec);
      const uint64_t own = c ? rec_inner(rec) + leb_bytes((uint64_t)(f - prev)) : 0u;
      const uint64_t bx = wave_incl_sum(own, lane) - own;
      if (in) {
        const uint64_t eo = eg + (x - c), bo = bg + bx;
        if (t == d.first_tile) {
          for (uint32_t s = d.off_lo; s <= d.slot; ++s) {
            if (a.d_tensor_offsets) a.d_tensor_offsets[s] = eo;
            if (a.d_tensor_byte_offsets) a.d_tensor_byte_offsets[s] = bo;
          }
        }
        if (t == a.num_tiles - 1) {
          for (uint32_t s = d.slot + 1; s <= a.num_tensors; ++s) {
            if (a.d_tensor_offsets) a.d_tensor_offsets[s] = eo + c;
            if (a.d_tensor_byte_offsets) a.d_tensor_byte_offsets[s] = bo + own;
          }
        }
      }
    }
  }
  __syncthreads();
  if (kOwnScan) {
    eg = sg.eg;
    bg = sg.bg;
  }
  const uint32_t total = sg.begin[64];
  // the last group's workgroup leaves the call's totals (own scan)
  auto finish = [&](uint64_t written) {
    if (kOwnScan && g == groups - 1 && threadIdx.x == 0) {
      *a.d_count = eg + total;
      *a.d_nbytes = bg + written;
    }
  };
  uint64_t written = 0;
  if (!sg.overflow) {
    for (uint32_t w0 = 0; w0 < total; w0 += kCodeWin) {
      const uint32_t n = total - w0 < (uint32_t)kCodeWin ? total - w0 : (uint32_t)kCodeWin;
      uint32_t v[kCodePer];
#pragma unroll
      for (int k = 0; k < kCodePer; ++k) {
        const uint32_t j = threadIdx.x + kThreads * k;
        uint32_t lo = 0, hi = kTilesPerGroup;
#pragma unroll
        for (int step = 0; step < 6; ++step) {
          const uint32_t mid = (lo + hi) >> 1;
          if (sg.begin[mid] <= w0 + j) lo = mid; else hi = mid;
        }
        v[k] = j < n ? __builtin_nontemporal_load(a.stage + (t0 + lo) * a.stage_stride +
                                                  (w0 + j - sg.begin[lo]))
                     : 0u;
      }
#pragma unroll
      for (int k = 0; k < kCodePer; ++k) {
        const uint32_t j = threadIdx.x + kThreads * k;
        if (j < n) sg.win[wslot(j)] = v[k];
      }
      __syncthreads();
      written += code_window(a, sg, w0, n, eg, bg, written);
    }
    finish(written);
    return;
  }
  for (uint32_t i = 0; i < n_here; ++i) {
    const uint32_t c = sg.count[i];
    if (c == 0) continue;
    const uint64_t tile = t0 + i;
    if (c <= a.stage_cap) {
      const uint32_t* slot = a.stage + tile * a.stage_stride;
      for (uint32_t r0 = 0; r0 < c; r0 += kCodeWin) {
        const uint32_t n = c - r0 < (uint32_t)kCodeWin ? c - r0 : (uint32_t)kCodeWin;
        for (uint32_t j = threadIdx.x; j < n; j += kThreads) sg.win[wslot(j)] = slot[r0 + j];
        __syncthreads();
        written += code_window(a, sg, sg.begin[i] + r0, n, eg, bg, written);
      }
      continue;
    }
    // an overflowed tile: read again for every window (a rare path; the
    // tile's registers are not kept across the windows)
    const TensorDesc d = tile_desc<kMulti>(a, tile);
    const uint32_t lane_word = (wave * kGroupsPerWave + lane) * 8;
    for (uint32_t r0 = 0; r0 < c; r0 += kCodeWin) {
      const uint32_t n = c - r0 < (uint32_t)kCodeWin ? c - r0 : (uint32_t)kCodeWin;
      TileScan s;
      scan_tile<kVec>(d, tile, lane, wave, s_wave_total, s);
#pragma unroll
      for (int u = 0; u < kChunks; ++u) {
        uint32_t m = s.mask[u];
        uint32_t r = s.rank[u];
        const uint32_t w0 = lane_word + 512 * u;
        while (m) {
          const int j = __builtin_ctz(m);
          m &= m - 1;
          if (r >= r0 && r < r0 + n) sg.win[wslot(r - r0)] = ((uint32_t)word_of(s.q[u], j) << 16) | (w0 + j);
          ++r;
        }
      }
      __syncthreads();
      written += code_window(a, sg, sg.begin[i] + r0, n, eg, bg, written);
    }
  }
  finish(written);
}

// ------------------------------------------------------- small kernels

__global__ void reset_kernel(uint64_t* d_count, uint64_t* d_offsets, uint32_t num_offsets) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  const uint64_t i0 = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (d_offsets)
    for (uint64_t i = i0; i < num_offsets; i += stride) d_offsets[i] = 0;
  if (i0 == 0) *d_count = 0;
}

__global__ void upload_words_kernel(WordBatch b, uint64_t* dst) {
  for (uint32_t i = threadIdx.x; i < b.count; i += blockDim.x) dst[i] = b.w[i];
}

// Row t of the table fills its tiles' map entries; a row's tiles are spread
// over gridDim.y workgroups (the largest tensors span tens of thousands).
__global__ void build_tile_map_kernel(const TensorDesc* table, uint32_t* tile_map) {
  const uint32_t t = blockIdx.x;
  const TensorDesc d = table[t];
  const uint64_t nt = tiles_for(d.n, d.head);
  const uint64_t stride = (uint64_t)gridDim.y * blockDim.x;
  for (uint64_t i = (uint64_t)blockIdx.y * blockDim.x + threadIdx.x; i < nt; i += stride)
    tile_map[d.first_tile + i] = t;
}

hipError_t launch_reset(uint64_t* d_count, uint64_t* d_offsets, uint32_t num_offsets,
                        hipStream_t stream) {
  uint64_t blocks = ((uint64_t)num_offsets + 255) / 256;
  if (blocks < 1) blocks = 1;
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(reset_kernel, dim3((uint32_t)blocks), dim3(256), 0, stream, d_count,
                     d_offsets, num_offsets);
  return hipGetLastError();
}

hipError_t launch_upload_words(const uint64_t* host_words, size_t nwords, uint64_t* dst,
                               hipStream_t stream) {
  for (size_t off = 0; off < nwords; off += kWordBatch) {
    WordBatch b;
    b.count = (nwords - off < (size_t)kWordBatch) ? nwords - off : kWordBatch;
    for (uint64_t i = 0; i < b.count; ++i) b.w[i] = host_words[off + i];
    hipLaunchKernelGGL(upload_words_kernel, dim3(1), dim3(256), 0, stream, b, dst + off);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_build_tile_map(const TensorDesc* table, uint32_t num_tensors,
                                 uint32_t* tile_map, hipStream_t stream) {
  if (num_tensors == 0) return hipSuccess;
  hipLaunchKernelGGL(build_tile_map_kernel, dim3(num_tensors, 8), dim3(256), 0, stream, table,
                     tile_map);
  return hipGetLastError();
}

template <typename CountT>
static hipError_t launch_group_scan_t(const CountT* counts, uint64_t num_tiles,
                                      uint64_t* group_sum, uint64_t* group_excl,
                                      uint64_t* d_total, hipStream_t stream) {
  const uint64_t groups = groups_for(num_tiles);
  if (groups <= kSmallScanGroups) {
    hipLaunchKernelGGL(tile_scan_kernel<CountT>, dim3(1), dim3(kScanThreads), 0, stream, counts,
                       num_tiles, group_excl, d_total);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(group_sum_kernel<CountT>, dim3((uint32_t)groups), dim3(64), 0, stream,
                     counts, num_tiles, group_sum);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(group_scan_kernel, dim3(1), dim3(kScanThreads), 0, stream, group_sum, groups,
                     group_excl, d_total);
  return hipGetLastError();
}

hipError_t launch_group_scan(const uint32_t* counts, uint64_t num_tiles, uint64_t* group_sum,
                             uint64_t* group_excl, uint64_t* d_total, hipStream_t stream) {
  return launch_group_scan_t(counts, num_tiles, group_sum, group_excl, d_total, stream);
}

hipError_t launch_group_scan(const uint64_t* counts, uint64_t num_tiles, uint64_t* group_sum,
                             uint64_t* group_excl, uint64_t* d_total, hipStream_t stream) {
  return launch_group_scan_t(counts, num_tiles, group_sum, group_excl, d_total, stream);
}

static hipError_t split_after_stage(hipStream_t stream, const StageSplit* split,
                                    hipStream_t& rest);

template <typename IdxT, bool kMulti, bool kVec>
static hipError_t launch_all(const ExtractArgs& a, hipStream_t stream, const StageSplit* split) {
  const uint64_t groups = (a.num_tiles + kTilesPerGroup - 1) / kTilesPerGroup;
  hipError_t e = record_scan_event(0, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((stage_kernel<kMulti, kVec, false>), dim3((uint32_t)a.num_tiles),
                     dim3(kThreads), 0, stream, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = record_scan_event(1, stream);
  if (e != hipSuccess) return e;
  // one tensor over few tiles: each tile finalizes itself (two launches)
  if (!kMulti && !split && a.num_inline == 1 && !a.d_tensor_offsets &&
      a.num_tiles <= kSmallTiles) {
    hipLaunchKernelGGL((finalize_small_kernel<IdxT, kVec>), dim3((uint32_t)a.num_tiles),
                       dim3(kThreads), 0, stream, a);
    return hipGetLastError();
  }
  hipStream_t rest;
  if (e == hipSuccess) e = split_after_stage(stream, split, rest);
  if (e != hipSuccess) return e;
  if (groups <= kOwnScanGroups) {
    hipLaunchKernelGGL((finalize_kernel<IdxT, kMulti, kVec, true>), dim3((uint32_t)groups),
                       dim3(kThreads), 0, rest, a);
    return hipGetLastError();
  }
  e = launch_group_scan(a.counts, a.num_tiles, a.group_sum, a.group_excl, a.d_count, rest);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((finalize_kernel<IdxT, kMulti, kVec, false>), dim3((uint32_t)groups),
                     dim3(kThreads), 0, rest, a);
  return hipGetLastError();
}

// After the stage kernel: the stream that takes the remaining kernels.
static hipError_t split_after_stage(hipStream_t stream, const StageSplit* split,
                                    hipStream_t& rest) {
  rest = stream;
  if (!split) return hipSuccess;
  hipError_t e = hipEventRecord(split->staged, stream);
  if (e == hipSuccess && split->rest != stream) e = hipStreamWaitEvent(split->rest, split->staged, 0);
  rest = split->rest;
  return e;
}

template <bool kMulti, bool kVec>
static hipError_t launch_coded(const ExtractArgs& a, hipStream_t stream, const StageSplit* split) {
  const uint64_t groups = (a.num_tiles + kTilesPerGroup - 1) / kTilesPerGroup;
  hipLaunchKernelGGL((stage_kernel<kMulti, kVec, true>), dim3((uint32_t)a.num_tiles),
                     dim3(kThreads), 0, stream, a);
  hipError_t e = hipGetLastError();
  hipStream_t rest;
  if (e == hipSuccess) e = split_after_stage(stream, split, rest);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(coded_group_kernel, dim3((uint32_t)groups), dim3(64), 0, rest, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (groups <= kOwnScanGroups) {
    hipLaunchKernelGGL((finalize_coded_kernel<kMulti, kVec, true>), dim3((uint32_t)groups),
                       dim3(kThreads), 0, rest, a);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(coded_scan_kernel, dim3(1), dim3(kScanThreads), 0, rest, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((finalize_coded_kernel<kMulti, kVec, false>), dim3((uint32_t)groups),
                     dim3(kThreads), 0, rest, a);
  return hipGetLastError();
}

template <bool kMulti, bool kVec>
static hipError_t launch_count_t(const ExtractArgs& a, hipStream_t stream) {
  hipError_t e = record_scan_event(0, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((count_kernel<kMulti, kVec>), dim3((uint32_t)a.num_tiles), dim3(kThreads),
                     kCountLds, stream, a);
  e = hipGetLastError();
  if (e == hipSuccess) e = record_scan_event(1, stream);
  if (e != hipSuccess) return e;
  return launch_group_scan(a.counts, a.num_tiles, a.group_sum, a.group_excl, a.d_count, stream);
}

hipError_t launch_count(const ExtractArgs& a, bool all_vec, hipStream_t stream) {
  if (a.num_tiles == 0) return hipSuccess;
  if (a.table != nullptr)
    return all_vec ? launch_count_t<true, true>(a, stream) : launch_count_t<true, false>(a, stream);
  return all_vec ? launch_count_t<false, true>(a, stream) : launch_count_t<false, false>(a, stream);
}

hipError_t launch_extract_coded(const ExtractArgs& a, bool all_vec, hipStream_t stream,
                                const StageSplit* split) {
  hipStream_t rest;
  if (a.num_tiles == 0) return split_after_stage(stream, split, rest);
  if (a.table != nullptr)
    return all_vec ? launch_coded<true, true>(a, stream, split)
                   : launch_coded<true, false>(a, stream, split);
  return all_vec ? launch_coded<false, true>(a, stream, split)
                 : launch_coded<false, false>(a, stream, split);
}

template <typename IdxT, bool kMulti>
static hipError_t launch_vec(const ExtractArgs& a, bool vec, hipStream_t stream,
                             const StageSplit* split) {
  return vec ? launch_all<IdxT, kMulti, true>(a, stream, split)
             : launch_all<IdxT, kMulti, false>(a, stream, split);
}

hipError_t launch_extract(const ExtractArgs& a, bool idx64, bool all_vec, hipStream_t stream,
                          const StageSplit* split) {
  hipStream_t rest;
  if (a.num_tiles == 0) return split_after_stage(stream, split, rest);
  const bool multi = a.table != nullptr;
  if (idx64)
    return multi ? launch_vec<int64_t, true>(a, all_vec, stream, split)
                 : launch_vec<int64_t, false>(a, all_vec, stream, split);
  return multi ? launch_vec<int32_t, true>(a, all_vec, stream, split)
               : launch_vec<int32_t, false>(a, all_vec, stream, split);
}

}  // namespace aurora
