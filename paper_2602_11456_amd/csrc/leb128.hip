// Gap + unsigned LEB128 index encoding on gfx950 (AuroraRL Sec. 5.1,
// "Sparse encoding" and the figure "Delta checkpoint index encoding"): a
// sorted index stream keeps its first entry as-is and every later entry as
// the difference from its predecessor; each number is then written as
// unsigned LEB128 (7 payload bits per byte, least significant group first,
// high bit set on every byte except the last).
//
// A stream may consist of segments (one per tensor, as in the paper, where
// every tensor has its own index array): the first entry of segment s is
// stored as idx - base[s], i.e. as the tensor-local index.
//
// Encode: per tile of 4096 entries the LEB128 byte count is summed
// (enc_count), the tile counts are scanned in groups (the same group scan
// as extract), and enc_write writes each entry's bytes at its offset.
// Decode: per tile of 16 KiB the terminating bytes (high bit clear) are
// counted (dec_count), scanned, and dec_gap turns every terminating byte
// into its entry's gap; a prefix sum with per-segment restarts
// (gap_sum, group scan, prefix, seg_corr, seg_add) gives the indices.
#include "delta_internal.h"

namespace aurora {

constexpr int kLebThreads = 256;
constexpr int kEncPer = 16;                       // entries per thread
constexpr int kEncTile = kLebThreads * kEncPer;   // 4096 entries
constexpr int kDecPer = 64;                       // bytes per thread
constexpr int kDecTile = kLebThreads * kDecPer;   // 16 KiB
constexpr int kDecBack = 16;                      // bytes read before a tile (a number has <= 10)

__device__ __forceinline__ uint32_t lane_of() { return threadIdx.x & 63; }

__device__ __forceinline__ uint32_t leb_len(uint64_t v) {
  const uint32_t bits = 64 - __builtin_clzll(v | 1ull);
  return (bits + 6) / 7;
}

// Segment of entry k: the last s < num with offs[s] <= k (num == 0: one
// segment, based at base0).
__device__ __forceinline__ uint32_t seg_of(const LebSegs& g, uint64_t k) {
  if (g.num == 0) return 0;
  uint32_t lo = 0, hi = g.num;
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) >> 1;
    if (g.offs[mid] <= k) lo = mid; else hi = mid;
  }
  return lo;
}
__device__ __forceinline__ uint64_t seg_lo(const LebSegs& g, uint32_t s) {
  return g.num ? g.offs[s] : 0;
}
__device__ __forceinline__ uint64_t seg_hi(const LebSegs& g, uint32_t s) {
  return (g.num && s + 1 < g.num) ? g.offs[s + 1] : ~0ull;
}
__device__ __forceinline__ int64_t seg_base(const LebSegs& g, uint32_t s) {
  return g.num ? (int64_t)g.bases[s] : g.base0;
}

// Exclusive prefix of v over the workgroup (kLebThreads threads) and the
// total.  Contains barriers; s_wave has kLebThreads / 64 entries.
template <typename T>
__device__ __forceinline__ T block_excl_scan(T v, T* s_wave, T& total) {
  const uint32_t lane = lane_of(), wave = threadIdx.x >> 6;
  T x = v;
#pragma unroll
  for (int s = 1; s < 64; s <<= 1) {
    const T y = __shfl_up(x, s);
    if ((int)lane >= s) x += y;
  }
  if (lane == 63) s_wave[wave] = x;
  __syncthreads();
  T before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kLebThreads / 64; ++w) {
    const T t = s_wave[w];
    before += (w < (int)wave) ? t : (T)0;
    all += t;
  }
  __syncthreads();
  total = all;
  return before + x - v;
}

// Sum of counts[g * kTilesPerGroup .. tile) (tiles before `tile` in its
// group), by wavefront 0; valid in thread 0... broadcast through LDS.
template <typename T>
__device__ __forceinline__ uint64_t group_before(const T* counts, uint64_t tile, uint64_t* s_out) {
  if (threadIdx.x < 64) {
    const uint64_t g0 = tile / kTilesPerGroup * kTilesPerGroup;
    const uint64_t t = g0 + threadIdx.x;
    uint64_t c = t < tile ? (uint64_t)counts[t] : 0;
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) c += __shfl_xor(c, s);
    if (threadIdx.x == 0) *s_out = c;
  }
  __syncthreads();
  return *s_out;
}

// ---------------------------------------------------------------- encode

// Gaps of the thread's kEncPer consecutive entries; returns their LEB128
// byte count.  s_idx holds the tile's entries with the entry before the
// tile at s_idx[0].
__device__ __forceinline__ uint32_t enc_gaps(const EncArgs& a, uint64_t t0, const int64_t* s_idx,
                                             uint64_t (&gap)[kEncPer], bool& bad) {
  const uint64_t k0 = t0 + (uint64_t)threadIdx.x * kEncPer;
  uint32_t bytes = 0;
  if (k0 >= a.count) {
#pragma unroll
    for (int j = 0; j < kEncPer; ++j) gap[j] = 0;
    return 0;
  }
  uint32_t sg = seg_of(a.segs, k0);
  uint64_t hi = seg_hi(a.segs, sg);
#pragma unroll
  for (int j = 0; j < kEncPer; ++j) {
    const uint64_t k = k0 + j;
    gap[j] = 0;
    if (k >= a.count) continue;
    while (k >= hi) {   // next segment (skips empty ones)
      ++sg;
      hi = seg_hi(a.segs, sg);
    }
    const int64_t cur = s_idx[k - t0 + 1];
    int64_t d;
    if (k == seg_lo(a.segs, sg)) {
      d = cur - seg_base(a.segs, sg);
      bad |= d < 0;
    } else {
      d = cur - s_idx[k - t0];
      bad |= d < 1;
    }
    gap[j] = d < 0 ? 0 : (uint64_t)d;
    bytes += leb_len(gap[j]);
  }
  return bytes;
}

__device__ __forceinline__ void enc_load_tile(const EncArgs& a, uint64_t t0, int64_t* s_idx) {
  for (uint32_t i = threadIdx.x; i < kEncTile + 1; i += kLebThreads) {
    // s_idx[i] = idx[t0 + i - 1]
    int64_t v = 0;
    if (i > 0 || t0 > 0) {
      const uint64_t k = t0 + i - 1;
      if (k < a.count) v = a.idx[k];
    }
    s_idx[i] = v;
  }
  __syncthreads();
}

__global__ __launch_bounds__(kLebThreads) void enc_count_kernel(EncArgs a) {
  __shared__ int64_t s_idx[kEncTile + 1];
  __shared__ uint32_t s_wave[kLebThreads / 64];
  const uint64_t tile = blockIdx.x;
  const uint64_t t0 = tile * kEncTile;
  enc_load_tile(a, t0, s_idx);
  uint64_t gap[kEncPer];
  bool bad = false;
  const uint32_t bytes = enc_gaps(a, t0, s_idx, gap, bad);
  uint32_t total;
  block_excl_scan(bytes, s_wave, total);
  if (threadIdx.x == 0) a.tile_bytes[tile] = total;
  if (bad && a.err)
    __hip_atomic_fetch_or(a.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ __launch_bounds__(kLebThreads) void enc_write_kernel(EncArgs a) {
  __shared__ int64_t s_idx[kEncTile + 1];
  __shared__ uint32_t s_wave[kLebThreads / 64];
  __shared__ uint64_t s_before;
  const uint64_t tile = blockIdx.x;
  const uint64_t t0 = tile * kEncTile;
  enc_load_tile(a, t0, s_idx);
  uint64_t gap[kEncPer];
  bool bad = false;
  const uint32_t bytes = enc_gaps(a, t0, s_idx, gap, bad);
  uint32_t total;
  const uint32_t excl = block_excl_scan(bytes, s_wave, total);
  const uint64_t tile_pos =
      a.group_excl[tile / kTilesPerGroup] + group_before(a.tile_bytes, tile, &s_before);
  uint64_t pos = tile_pos + excl;
  const uint64_t k0 = t0 + (uint64_t)threadIdx.x * kEncPer;
  uint32_t sg = k0 < a.count ? seg_of(a.segs, k0) : 0;
  uint64_t hi = seg_hi(a.segs, sg);
#pragma unroll
  for (int j = 0; j < kEncPer; ++j) {
    const uint64_t k = k0 + j;
    if (k >= a.count) break;
    while (k >= hi) {
      ++sg;
      hi = seg_hi(a.segs, sg);
    }
    if (a.seg_byte_offsets && a.segs.num && k == seg_lo(a.segs, sg)) {
      // this entry opens segment sg and every empty segment just before it
      for (int64_t s = sg; s >= 0 && a.segs.offs[s] == k; --s) a.seg_byte_offsets[s] = pos;
    }
    uint64_t v = gap[j];
    do {
      uint8_t b = (uint8_t)(v & 0x7F);
      v >>= 7;
      if (v) b |= 0x80;
      if (pos < a.capacity) a.out[pos] = b;
      ++pos;
    } while (v);
  }
}

// Segments that open at or after the last entry (and the end slot) start
// at the total byte count.
__global__ void enc_seg_tail_kernel(EncArgs a) {
  const uint64_t total = *a.d_nbytes;
  for (uint32_t s = threadIdx.x + blockIdx.x * blockDim.x; s <= a.segs.num;
       s += blockDim.x * gridDim.x) {
    if (s == a.segs.num || a.segs.offs[s] >= a.count) a.seg_byte_offsets[s] = total;
  }
}

// ---------------------------------------------------------------- decode

__device__ __forceinline__ void dec_load_tile(const DecArgs& a, uint64_t b0, uint8_t* s_bytes) {
  // s_bytes[i] = in[b0 - kDecBack + i] for i < kDecBack + kDecTile (0 outside)
  for (uint32_t i = threadIdx.x; i < kDecBack + kDecTile; i += kLebThreads) {
    const int64_t p = (int64_t)b0 - kDecBack + (int64_t)i;
    s_bytes[i] = (p >= 0 && (uint64_t)p < a.nbytes) ? a.in[p] : 0;
  }
  __syncthreads();
}

__global__ __launch_bounds__(kLebThreads) void dec_count_kernel(DecArgs a) {
  __shared__ uint32_t s_wave[kLebThreads / 64];
  const uint64_t tile = blockIdx.x;
  const uint64_t p0 = tile * kDecTile + (uint64_t)threadIdx.x * kDecPer;
  uint32_t c = 0;
  for (int i = 0; i < kDecPer; ++i) {
    const uint64_t p = p0 + i;
    if (p < a.nbytes && (a.in[p] & 0x80) == 0) ++c;
  }
  uint32_t total;
  block_excl_scan(c, s_wave, total);
  if (threadIdx.x == 0) a.tile_terms[tile] = total;
}

// Every terminating byte gives one entry's gap: its number runs from the
// byte after the previous terminating byte up to it.
__global__ __launch_bounds__(kLebThreads) void dec_gap_kernel(DecArgs a) {
  __shared__ uint8_t s_bytes[kDecBack + kDecTile];
  __shared__ uint32_t s_wave[kLebThreads / 64];
  __shared__ uint64_t s_before;
  const uint64_t tile = blockIdx.x;
  const uint64_t b0 = tile * kDecTile;
  dec_load_tile(a, b0, s_bytes);
  const uint32_t q0 = threadIdx.x * kDecPer;   // thread's first byte in the tile
  uint32_t c = 0;
  for (int i = 0; i < kDecPer; ++i) {
    const uint64_t p = b0 + q0 + i;
    if (p < a.nbytes && (s_bytes[kDecBack + q0 + i] & 0x80) == 0) ++c;
  }
  uint32_t total;
  const uint32_t excl = block_excl_scan(c, s_wave, total);
  uint64_t e = a.group_excl[tile / kTilesPerGroup] + group_before(a.tile_terms, tile, &s_before) +
               excl;
  bool bad = false;
  for (int i = 0; i < kDecPer; ++i) {
    const uint64_t p = b0 + q0 + i;
    if (p >= a.nbytes) break;
    const uint32_t li = kDecBack + q0 + i;
    if (s_bytes[li] & 0x80) {
      if (p == a.nbytes - 1) bad = true;   // the stream ends inside a number
      continue;
    }
    // bytes of this number: li - len + 1 .. li
    uint32_t len = 1;
    while (len <= 10 && li >= len && p >= len && (s_bytes[li - len] & 0x80)) ++len;
    uint64_t v = 0;
    if (len > 10) {
      bad = true;
    } else {
      for (uint32_t m = 0; m < len; ++m) {
        const uint64_t payload = s_bytes[li - len + 1 + m] & 0x7F;
        if (m == 9 && payload > 1) bad = true;   // more than 64 bits
        v |= payload << (7 * m);
      }
    }
    if (e < a.capacity) a.out[e] = (int64_t)v;
    ++e;
  }
  if (bad && a.err)
    __hip_atomic_fetch_or(a.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Number of decoded entries that are in the output.
__device__ __forceinline__ uint64_t dec_kept(const DecArgs& a) {
  const uint64_t n = *a.d_count;
  return n < a.capacity ? n : a.capacity;
}

__global__ __launch_bounds__(kLebThreads) void gap_sum_kernel(DecArgs a) {
  __shared__ uint64_t s_wave[kLebThreads / 64];
  const uint64_t K = dec_kept(a);
  const uint64_t k0 = (uint64_t)blockIdx.x * kEncTile + (uint64_t)threadIdx.x * kEncPer;
  uint64_t sum = 0;
#pragma unroll
  for (int j = 0; j < kEncPer; ++j)
    if (k0 + j < K) sum += (uint64_t)a.out[k0 + j];
  uint64_t total;
  block_excl_scan(sum, s_wave, total);
  if (threadIdx.x == 0) a.sum_tile[blockIdx.x] = total;
}

// In place: out[k] = gap[0] + ... + gap[k].
__global__ __launch_bounds__(kLebThreads) void prefix_kernel(DecArgs a) {
  __shared__ uint64_t s_wave[kLebThreads / 64];
  __shared__ uint64_t s_before;
  const uint64_t K = dec_kept(a);
  const uint64_t tile = blockIdx.x;
  const uint64_t k0 = tile * kEncTile + (uint64_t)threadIdx.x * kEncPer;
  uint64_t g[kEncPer];
  uint64_t sum = 0;
#pragma unroll
  for (int j = 0; j < kEncPer; ++j) {
    g[j] = (k0 + j < K) ? (uint64_t)a.out[k0 + j] : 0;
    sum += g[j];
  }
  uint64_t total;
  const uint64_t excl = block_excl_scan(sum, s_wave, total);
  uint64_t run = a.sum_group_excl[tile / kTilesPerGroup] +
                 group_before(a.sum_tile, tile, &s_before) + excl;
#pragma unroll
  for (int j = 0; j < kEncPer; ++j) {
    run += g[j];
    if (k0 + j < K) a.out[k0 + j] = (int64_t)run;
  }
}

// corr[s] = base[s] - (prefix just before segment s).
__global__ void seg_corr_kernel(DecArgs a) {
  const uint64_t K = dec_kept(a);
  for (uint32_t s = threadIdx.x + blockIdx.x * blockDim.x; s < a.segs.num;
       s += blockDim.x * gridDim.x) {
    const uint64_t o = a.segs.offs[s];
    const int64_t before = (o > 0 && o - 1 < K) ? a.out[o - 1] : 0;
    a.corr[s] = (int64_t)a.segs.bases[s] - before;
  }
}

__global__ __launch_bounds__(kLebThreads) void seg_add_kernel(DecArgs a) {
  const uint64_t K = dec_kept(a);
  const uint64_t k0 = (uint64_t)blockIdx.x * kEncTile + (uint64_t)threadIdx.x * kEncPer;
  if (k0 >= K) return;
  uint32_t sg = seg_of(a.segs, k0);
  uint64_t hi = seg_hi(a.segs, sg);
#pragma unroll
  for (int j = 0; j < kEncPer; ++j) {
    const uint64_t k = k0 + j;
    if (k >= K) break;
    while (k >= hi) {
      ++sg;
      hi = seg_hi(a.segs, sg);
    }
    a.out[k] += a.corr[sg];
  }
}

// --------------------------------------------------------------- launches

static uint64_t enc_tiles(uint64_t count) { return (count + kEncTile - 1) / kEncTile; }
static uint64_t dec_tiles(uint64_t nbytes) { return (nbytes + kDecTile - 1) / kDecTile; }

EncLayout enc_layout(uint64_t count) {
  EncLayout L;
  const uint64_t tiles = enc_tiles(count), groups = groups_for(tiles);
  L.tiles = tiles;
  L.tile_bytes = 0;
  L.group_sum = align_up(4 * tiles);
  L.group_excl = align_up(L.group_sum + 8 * groups);
  L.total = align_up(L.group_excl + 8 * groups);
  return L;
}

DecLayout dec_layout(uint64_t nbytes, uint64_t capacity, uint32_t num_segs) {
  DecLayout L;
  const uint64_t bt = dec_tiles(nbytes);
  const uint64_t kmax = nbytes < capacity ? nbytes : capacity;   // an entry takes >= 1 byte
  const uint64_t et = enc_tiles(kmax);
  L.btiles = bt;
  L.etiles = et;
  L.tile_terms = 0;
  L.group_sum = align_up(4 * bt);
  L.group_excl = align_up(L.group_sum + 8 * groups_for(bt));
  L.sum_tile = align_up(L.group_excl + 8 * groups_for(bt));
  L.sum_group_sum = align_up(L.sum_tile + 8 * et);
  L.sum_group_excl = align_up(L.sum_group_sum + 8 * groups_for(et));
  L.sum_total = align_up(L.sum_group_excl + 8 * groups_for(et));
  L.corr = align_up(L.sum_total + 8);
  L.total = align_up(L.corr + 8 * (uint64_t)num_segs);
  return L;
}

hipError_t launch_leb128_encode(EncArgs a, uint64_t* group_sum, uint64_t* group_excl,
                                hipStream_t stream) {
  const uint64_t tiles = enc_tiles(a.count);
  hipError_t e;
  if (tiles == 0) {
    e = launch_reset(a.d_nbytes, nullptr, 0, stream);
  } else {
    hipLaunchKernelGGL(enc_count_kernel, dim3((uint32_t)tiles), dim3(kLebThreads), 0, stream, a);
    e = hipGetLastError();
    if (e == hipSuccess)
      e = launch_group_scan(a.tile_bytes, tiles, group_sum, group_excl, a.d_nbytes, stream);
    a.group_excl = group_excl;
    if (e == hipSuccess) {
      hipLaunchKernelGGL(enc_write_kernel, dim3((uint32_t)tiles), dim3(kLebThreads), 0, stream, a);
      e = hipGetLastError();
    }
  }
  if (e == hipSuccess && a.seg_byte_offsets) {
    const uint32_t n = a.segs.num + 1;
    hipLaunchKernelGGL(enc_seg_tail_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, a);
    e = hipGetLastError();
  }
  return e;
}

hipError_t launch_leb128_decode(DecArgs a, const DecLayout& L, char* ws, hipStream_t stream) {
  hipError_t e;
  if (L.btiles == 0) return launch_reset(a.d_count, nullptr, 0, stream);
  uint64_t* gs = (uint64_t*)(ws + L.group_sum);
  a.group_excl = (uint64_t*)(ws + L.group_excl);
  a.sum_tile = (uint64_t*)(ws + L.sum_tile);
  a.sum_group_excl = (uint64_t*)(ws + L.sum_group_excl);
  a.corr = (int64_t*)(ws + L.corr);
  hipLaunchKernelGGL(dec_count_kernel, dim3((uint32_t)L.btiles), dim3(kLebThreads), 0, stream, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if ((e = launch_group_scan(a.tile_terms, L.btiles, gs, a.group_excl, a.d_count, stream)) !=
      hipSuccess)
    return e;
  hipLaunchKernelGGL(dec_gap_kernel, dim3((uint32_t)L.btiles), dim3(kLebThreads), 0, stream, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (L.etiles == 0) return hipSuccess;
  hipLaunchKernelGGL(gap_sum_kernel, dim3((uint32_t)L.etiles), dim3(kLebThreads), 0, stream, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if ((e = launch_group_scan(a.sum_tile, L.etiles, (uint64_t*)(ws + L.sum_group_sum),
                             a.sum_group_excl, (uint64_t*)(ws + L.sum_total), stream)) !=
      hipSuccess)
    return e;
  hipLaunchKernelGGL(prefix_kernel, dim3((uint32_t)L.etiles), dim3(kLebThreads), 0, stream, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (a.segs.num == 0) return hipSuccess;
  hipLaunchKernelGGL(seg_corr_kernel, dim3((a.segs.num + 255) / 256), dim3(256), 0, stream, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(seg_add_kernel, dim3((uint32_t)L.etiles), dim3(kLebThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace aurora
