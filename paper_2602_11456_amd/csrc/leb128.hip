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
// Encode, per tile of 4096 entries (one workgroup, each wavefront 1024
// consecutive entries, 64 per step, so every load is coalesced): enc_stage
// reads the indices once and stages each tile's code (wavefront scan of
// the code lengths per step) with its byte count; the byte counts are
// scanned in groups (the same group scan as extract), and enc_copy moves
// every tile's code to its place.
//
// Decode, per tile of 16 KiB of bytes: dec_count counts the terminating
// bytes (high bit clear; 4 bytes per 32-bit test); their scan numbers the
// entries.  dec_fold decodes every number (a terminating byte and the
// continuation bytes before it, at most 10) and folds the tile into a
// segmented sum: an entry that opens a segment contributes base + term and
// restarts the sum, any other adds its gap.  Those tile folds are scanned
// (segmented), and dec_write decodes again and writes every index as the
// segmented running sum.
#include "delta_internal.h"
#include "leb128.h"

namespace aurora {

constexpr int kLebThreads = 256;
constexpr int kLebWaves = kLebThreads / 64;
constexpr int kEncSteps = 16;                    // 64-entry steps per wavefront
constexpr int kEncWave = 64 * kEncSteps;         // 1024 entries
constexpr int kEncTile = kLebWaves * kEncWave;   // 4096 entries
constexpr int kDecWave = 4096;                   // bytes per wavefront
constexpr int kDecTile = kLebWaves * kDecWave;   // 16 KiB
constexpr int kDecBack = 16;                     // bytes kept before a tile (>= 9)
constexpr int kSegLds = 256;                     // segment starts cached per tile

__device__ __forceinline__ uint32_t lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ uint32_t wave_id() { return threadIdx.x >> 6; }

__device__ __forceinline__ uint32_t leb_len(uint64_t v) {
  const uint32_t bits = 64 - __builtin_clzll(v | 1ull);
  return (bits + 6) / 7;
}

__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) v += __shfl_xor(v, s);
  return v;
}

template <typename T>
__device__ __forceinline__ T wave_incl_scan(T v) {
  const uint32_t lane = lane_id();
#pragma unroll
  for (int s = 1; s < 64; s <<= 1) {
    const T y = __shfl_up(v, s);
    if ((int)lane >= s) v += y;
  }
  return v;
}

// Segmented inclusive scan over the wavefront: a lane with f set restarts
// the running sum at its own v.
__device__ __forceinline__ void wave_seg_scan(uint32_t& f, uint64_t& v) {
  const uint32_t lane = lane_id();
#pragma unroll
  for (int s = 1; s < 64; s <<= 1) {
    const uint64_t vp = __shfl_up(v, s);
    const uint32_t fp = __shfl_up(f, s);
    if ((int)lane >= s) {
      if (!f) v += vp;
      f |= fp;
    }
  }
}

// ------------------------------------------------------------- segments

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
// base0 as a value with no address: otherwise the compiler may merge the
// two reads of a base into one load through a pointer chosen between
// base0 and bases[s], which needs base0 in (slow) scratch memory.
__device__ __forceinline__ int64_t seg_base0(const LebSegs& g) {
  int64_t b = g.base0;
  __asm__ volatile("" : "+v"(b));
  return b;
}
__device__ __forceinline__ int64_t seg_base(const LebSegs& g, uint32_t s) {
  return g.num ? (int64_t)g.bases[s] : seg_base0(g);
}

// The segments that a tile's entries fall in: first..last, with their
// starts cached in LDS when there are few (from the tile's record, written
// by enc_segs_kernel or dec_recs_kernel).
struct TileSegs {
  uint32_t first, last;
  bool cached;
  uint64_t lo0;   // first entry of segment `first`
};

// Segment of entry e of the tile, and whether e opens it (entry 0 always
// opens the first segment).
__device__ __forceinline__ uint32_t tile_seg(const LebSegs& g, const TileSegs& c,
                                             const uint64_t* s_lo, uint64_t e, bool& start) {
  if (g.num == 0) {
    start = e == 0;
    return 0;
  }
  uint32_t s;
  uint64_t lo;
  if (c.first == c.last) {
    s = c.first;
    lo = c.lo0;
  } else if (c.cached) {
    uint32_t a = 0, b = c.last - c.first + 1;
    while (b - a > 1) {
      const uint32_t mid = (a + b) >> 1;
      if (s_lo[mid] <= e) a = mid; else b = mid;
    }
    s = c.first + a;
    lo = s_lo[a];
  } else {
    s = seg_of(g, e);
    lo = g.offs[s];
  }
  start = e == 0 || e == lo;
  return s;
}

__device__ __forceinline__ void raise_flag(uint32_t* err) {
  if (err) __hip_atomic_fetch_or(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------- encode
//
// One read of the indices.  enc_stage: per tile, the gaps and their code
// lengths, a wavefront scan of the lengths per step, the tile's bytes
// assembled in LDS and stored to the tile's staging slot (16-byte stores),
// its byte count, and the tile-local byte offset of every segment that
// opens in it.  The byte counts are scanned in groups.  enc_copy: every
// tile's staged bytes to their place in the output; a tile whose code
// outgrew its slot is encoded again straight to the output.  enc_seg_fix
// makes the segment byte offsets absolute.  Traffic per index: 8 bytes
// read once, its code written, read and written again (about 1.3 bytes
// each at 1% density), where counting and then writing read the indices
// twice.

constexpr int kEncLds = 16384;                  // LDS assembly area of a tile's code
constexpr uint32_t kEncSlot = 2 * kEncTile;     // staged code bytes per tile
static_assert(kEncSlot <= (uint32_t)kEncLds && kEncSlot % 16 == 0, "encoder slot size");
typedef uint32_t enc_u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint64_t enc_count_of(const EncArgs& a) {
  if (!a.d_count_in) return a.count;
  const uint64_t c = *a.d_count_in;
  return c < a.count ? c : a.count;
}

// This lane's indices kw + 64 it (it < kEncSteps) below t1, and the index
// just before the wavefront's first entry (0 for the stream's first).
struct EncLoad {
  int64_t cur[kEncSteps];
  int64_t last;
};

__device__ __forceinline__ void enc_load(const EncArgs& a, uint64_t kw, uint64_t t1, EncLoad& L) {
  const uint32_t lane = lane_id();
#pragma unroll
  for (int it = 0; it < kEncSteps; ++it) {
    const uint64_t k = kw + 64 * it;
    L.cur[it] = k < t1 ? a.idx[k] : 0;
  }
  const uint64_t first = kw - lane;   // the wavefront's first entry
  L.last = (first > 0 && first < t1) ? a.idx[first - 1] : 0;
}

// Gaps of the loaded entries: idx - base for an entry that opens its
// segment, else idx - previous idx (the previous index comes from the
// neighbouring lane).  Sets bit it of `starts` for an entry that opens a
// segment, `bad` for a gap below 0 / 1; returns the lane's code bytes.
// The gaps replace the indices in L.cur (each step reads its own index, and
// its neighbour's through a shuffle, before writing the gap).
__device__ __forceinline__ uint32_t enc_gaps(const EncArgs& a, const TileSegs& c,
                                             const uint64_t* s_lo, uint64_t kw, uint64_t t1,
                                             EncLoad& L, uint32_t& starts, bool& bad) {
  const uint32_t lane = lane_id();
  int64_t last = L.last;
  uint32_t bytes = 0;
  starts = 0;
#pragma unroll
  for (int it = 0; it < kEncSteps; ++it) {
    const uint64_t k = kw + 64 * it;
    const int64_t cur = L.cur[it];
    int64_t prev = __shfl_up(cur, 1);
    if (lane == 0) prev = last;
    last = __shfl(cur, 63);
    uint64_t g = 0;
    if (k < t1) {
      bool start;
      const uint32_t seg = tile_seg(a.segs, c, s_lo, k, start);
      int64_t d;
      if (start) {
        d = cur - seg_base(a.segs, seg);
        bad |= d < 0;
      } else {
        d = cur - prev;
        bad |= d < 1;
      }
      g = d < 0 ? 0 : (uint64_t)d;
      starts |= (uint32_t)start << it;
      bytes += leb_len(g);
    }
    L.cur[it] = (int64_t)g;
  }
  return bytes;
}

// Position of every entry's code inside the tile (wavefront scans of the
// lengths, starting at `pos`, this wavefront's offset in the tile); calls
// f(it, k, len, p, gap) for each of the lane's entries inside the tile.
template <typename F>
__device__ __forceinline__ void enc_walk(uint64_t kw, uint64_t t1, const int64_t (&gap)[kEncSteps],
                                         uint32_t pos, F f) {
#pragma unroll
  for (int it = 0; it < kEncSteps; ++it) {
    const uint64_t k = kw + 64 * it;
    const uint64_t g = (uint64_t)gap[it];
    const uint32_t len = k < t1 ? leb_len(g) : 0;
    const uint32_t incl = wave_incl_scan(len);
    if (len) f(it, k, len, pos + incl - len, g);
    pos += __shfl(incl, 63);
  }
}

// The bytes of one number: 7 payload bits each, low group first.
template <typename Put>
__device__ __forceinline__ void enc_bytes(uint64_t v, uint32_t len, Put put) {
  for (uint32_t m = 0; m < len; ++m) {
    put(m, (uint8_t)((v & 0x7F) | (m + 1 < len ? 0x80u : 0u)));
    v >>= 7;
  }
}

// Segment range of every encoder tile (first and last segment of its
// entries, and the first entry of the first), one thread per tile, so that
// the tile's workgroups take it with one load instead of searching.
__global__ void enc_segs_kernel(EncArgs a) {
  const uint64_t count = enc_count_of(a);
  const uint64_t tiles = (count + kEncTile - 1) / kEncTile;
  for (uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; t < tiles;
       t += (uint64_t)gridDim.x * blockDim.x) {
    const uint64_t t0 = t * kEncTile;
    const uint64_t t1 = t0 + kEncTile < count ? t0 + kEncTile : count;
    const uint32_t first = seg_of(a.segs, t0), last = seg_of(a.segs, t1 - 1);
    a.tile_segs[t] = EncTileSegs{first, last, a.segs.offs[first]};
  }
}

// The tile's segments from its record (contains a barrier when it spans
// several segments, whose starts are then cached in LDS).
__device__ __forceinline__ TileSegs enc_tile_segs(const EncArgs& a, uint64_t tile,
                                                  uint64_t* s_lo) {
  TileSegs c{0, 0, false, 0};
  if (a.segs.num == 0) return c;
  const EncTileSegs r = a.tile_segs[tile];
  c.first = r.first;
  c.last = r.last;
  c.lo0 = r.lo0;
  const uint32_t n = c.last - c.first + 1;
  if (n > 1) {   // uniform
    if (n <= (uint32_t)kSegLds) {
      for (uint32_t j = threadIdx.x; j < n; j += kLebThreads) s_lo[j] = a.segs.offs[c.first + j];
      c.cached = true;
    }
    __syncthreads();
  }
  return c;
}

// Tiles loop grid-stride (the entry count may only be known on the device).
__global__ __launch_bounds__(kLebThreads) void enc_stage_kernel(EncArgs a) {
  __shared__ uint64_t s_lo[kSegLds];
  __shared__ uint32_t s_wave[kLebWaves];
  __shared__ __align__(16) uint8_t s_out[kEncSlot];
  const uint64_t count = enc_count_of(a);
  const uint64_t tiles = (count + kEncTile - 1) / kEncTile;
  const uint32_t lane = lane_id(), wave = wave_id();
  bool bad = false;
  for (uint64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
    const uint64_t t0 = tile * kEncTile;
    const uint64_t t1 = t0 + kEncTile < count ? t0 + kEncTile : count;
    const uint64_t kw = t0 + (uint64_t)wave * kEncWave + lane;
    EncLoad L;
    enc_load(a, kw, t1, L);
    const TileSegs c = enc_tile_segs(a, tile, s_lo);
    uint32_t starts;
    const uint32_t bytes = wave_sum(enc_gaps(a, c, s_lo, kw, t1, L, starts, bad));
    if (lane == 0) s_wave[wave] = bytes;
    __syncthreads();
    uint32_t pos = 0, total = 0;
#pragma unroll
    for (int w = 0; w < kLebWaves; ++w) {
      pos += (uint32_t)w < wave ? s_wave[w] : 0u;
      total += s_wave[w];
    }
    const bool staged = total <= kEncSlot;
    const bool segs_out = a.seg_byte_offsets && a.segs.num;
    enc_walk(kw, t1, L.cur, pos, [&](int it, uint64_t k, uint32_t len, uint32_t p, uint64_t v) {
      if (segs_out && ((starts >> it) & 1u)) {
        // this entry opens its segment and every empty one just before it:
        // their tile-local offset (made absolute by enc_seg_fix)
        bool st;
        const uint32_t sg = tile_seg(a.segs, c, s_lo, k, st);
        for (int64_t s = sg; s >= 0 && a.segs.offs[s] == k; --s) a.seg_byte_offsets[s] = p;
      }
      if (staged) enc_bytes(v, len, [&](uint32_t m, uint8_t b) { s_out[p + m] = b; });
    });
    __syncthreads();
    if (staged) {
      enc_u32x4* slot = (enc_u32x4*)(a.stage + tile * kEncSlot);
      const enc_u32x4* src = (const enc_u32x4*)s_out;
      for (uint32_t i = threadIdx.x; i < (total + 15) / 16; i += kLebThreads)
        __builtin_nontemporal_store(src[i], slot + i);
    }
    if (threadIdx.x == 0) a.tile_bytes[tile] = total;
    __syncthreads();   // s_out and s_wave are reused by the next tile
  }
  if (bad) raise_flag(a.err);
}

// Sums of the tile byte counts per group of kTilesPerGroup tiles (tiles
// past the entry count add nothing).
__global__ __launch_bounds__(64) void enc_group_sum_kernel(EncArgs a, uint64_t* group_sum) {
  const uint64_t tiles = (enc_count_of(a) + kEncTile - 1) / kEncTile;
  const uint64_t t = (uint64_t)blockIdx.x * kTilesPerGroup + lane_id();
  const uint64_t v = wave_sum(t < tiles ? (uint64_t)a.tile_bytes[t] : 0ull);
  if (lane_id() == 0) group_sum[blockIdx.x] = v;
}

// Stores bytes [0, n) of s_out at out + pos (4-byte stores where the
// destination is aligned).
__device__ __forceinline__ void enc_flush(const uint8_t* s_out, uint64_t n, uint8_t* out,
                                          uint64_t pos) {
  uint8_t* dst = out + pos;
  const uint64_t head = (4 - ((uintptr_t)dst & 3u)) & 3u;
  const uint64_t h = head < n ? head : n;
  const uint64_t words = (n - h) / 4;
  for (uint64_t i = threadIdx.x; i < h; i += kLebThreads) dst[i] = s_out[i];
  uint32_t* dw = (uint32_t*)(dst + h);
  for (uint64_t w = threadIdx.x; w < words; w += kLebThreads) {
    const uint64_t j = h + 4 * w;
    dw[w] = (uint32_t)s_out[j] | ((uint32_t)s_out[j + 1] << 8) | ((uint32_t)s_out[j + 2] << 16) |
            ((uint32_t)s_out[j + 3] << 24);
  }
  for (uint64_t i = h + 4 * words + threadIdx.x; i < n; i += kLebThreads) dst[i] = s_out[i];
}

__global__ __launch_bounds__(kLebThreads) void enc_copy_kernel(EncArgs a) {
  __shared__ uint64_t s_lo[kSegLds];
  __shared__ uint32_t s_wave[kLebWaves];
  __shared__ uint64_t s_before;
  __shared__ __align__(16) uint8_t s_out[kEncSlot];
  const uint64_t count = enc_count_of(a);
  const uint64_t tiles = (count + kEncTile - 1) / kEncTile;
  const uint32_t lane = lane_id(), wave = wave_id();
  for (uint64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
    // the tile's output position: its group's offset plus the byte counts
    // of the group's earlier tiles
    const uint64_t gt = tile / kTilesPerGroup * kTilesPerGroup + lane;
    const uint64_t before_part = (wave == 0 && gt < tile) ? (uint64_t)a.tile_bytes[gt] : 0;
    const uint64_t gexcl = a.group_excl[tile / kTilesPerGroup];
    const uint32_t total = a.tile_bytes[tile];
    if (wave == 0) {
      const uint64_t b = wave_sum(before_part);
      if (lane == 0) s_before = b;
    }
    if (total <= kEncSlot) {
      const enc_u32x4* slot = (const enc_u32x4*)(a.stage + tile * kEncSlot);
      enc_u32x4* dst = (enc_u32x4*)s_out;
      for (uint32_t i = threadIdx.x; i < (total + 15) / 16; i += kLebThreads)
        dst[i] = __builtin_nontemporal_load(slot + i);
    }
    __syncthreads();
    const uint64_t tile_pos = gexcl + s_before;
    const uint64_t room = a.capacity > tile_pos ? a.capacity - tile_pos : 0;
    if (total <= kEncSlot) {
      enc_flush(s_out, total < room ? total : room, a.out, tile_pos);
    } else {
      // the code outgrew the slot: encode the tile again, each entry's bytes
      // stored straight to the output
      const uint64_t t0 = tile * kEncTile;
      const uint64_t t1 = t0 + kEncTile < count ? t0 + kEncTile : count;
      const uint64_t kw = t0 + (uint64_t)wave * kEncWave + lane;
      EncLoad L;
      enc_load(a, kw, t1, L);
      const TileSegs c = enc_tile_segs(a, tile, s_lo);
      uint32_t starts;
      bool bad = false;   // reported by enc_stage
      const uint32_t bytes = wave_sum(enc_gaps(a, c, s_lo, kw, t1, L, starts, bad));
      if (lane == 0) s_wave[wave] = bytes;
      __syncthreads();
      uint32_t pos = 0;
#pragma unroll
      for (int w = 0; w < kLebWaves; ++w) pos += (uint32_t)w < wave ? s_wave[w] : 0u;
      enc_walk(kw, t1, L.cur, pos, [&](int, uint64_t, uint32_t len, uint32_t p, uint64_t v) {
        enc_bytes(v, len, [&](uint32_t m, uint8_t b) {
          if (tile_pos + p + m < a.capacity) a.out[tile_pos + p + m] = b;
        });
      });
    }
    __syncthreads();   // s_out, s_before and s_wave are reused by the next tile
  }
}

// Segment byte offsets: a segment that opens at entry k < count gets its
// tile's output position added to the tile-local offset enc_stage left;
// segments that open at or after the last entry (and the end slot) start
// at the total byte count.
__global__ void enc_seg_fix_kernel(EncArgs a) {
  const uint64_t total = *a.d_nbytes;
  const uint64_t count = enc_count_of(a);
  for (uint32_t s = threadIdx.x + blockIdx.x * blockDim.x; s <= a.segs.num;
       s += blockDim.x * gridDim.x) {
    if (s == a.segs.num || a.segs.offs[s] >= count) {
      a.seg_byte_offsets[s] = total;
      continue;
    }
    const uint64_t tile = a.segs.offs[s] / kEncTile;
    uint64_t pos = a.group_excl[tile / kTilesPerGroup];
    for (uint64_t t = tile / kTilesPerGroup * kTilesPerGroup; t < tile; ++t) pos += a.tile_bytes[t];
    a.seg_byte_offsets[s] += pos;
  }
}

// ---------------------------------------------------------------- decode

// Terminating bytes (high bit clear) among the 4 bytes of w whose
// positions p0 .. p0+3 are below n.
__device__ __forceinline__ uint32_t terms_in_word(uint32_t w, uint64_t p0, uint64_t n) {
  uint32_t m = ~w & 0x80808080u;
  if (p0 + 4 > n) m &= p0 >= n ? 0u : (0xFFFFFFFFu >> (8 * (4 - (n - p0))));
  return __builtin_popcount(m);
}

typedef uint32_t leb_u32x4 __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(1))) leb_u32x4* leb_gvec_ptr;

// The 16 bytes at p (16-aligned; bytes at or past n read as 0).
__device__ __forceinline__ uint4 load16(const uint8_t* in, uint64_t p, uint64_t n) {
  if (p + 16 <= n) {
    const leb_u32x4 v = __builtin_nontemporal_load((leb_gvec_ptr)(uintptr_t)(in + p));
    return {v.x, v.y, v.z, v.w};
  }
  uint32_t w[4] = {0u, 0u, 0u, 0u};
  for (uint32_t i = 0; i < 16 && p + i < n; ++i) w[i >> 2] |= (uint32_t)in[p + i] << (8 * (i & 3));
  return {w[0], w[1], w[2], w[3]};
}

__global__ __launch_bounds__(kLebThreads) void dec_count_kernel(DecArgs a, bool aligned) {
  __shared__ uint32_t s_wave[kLebWaves];
  const uint64_t b0 = (uint64_t)blockIdx.x * kDecTile;
  uint32_t c = 0;
  if (aligned) {
#pragma unroll
    for (int j = 0; j < kDecTile / 16 / kLebThreads; ++j) {
      const uint64_t p = b0 + 16ull * (j * kLebThreads + threadIdx.x);
      if (p < a.nbytes) {
        const uint4 v = load16(a.in, p, a.nbytes);
        c += terms_in_word(v.x, p, a.nbytes) + terms_in_word(v.y, p + 4, a.nbytes) +
             terms_in_word(v.z, p + 8, a.nbytes) + terms_in_word(v.w, p + 12, a.nbytes);
      }
    }
  } else {
    for (uint32_t i = threadIdx.x; i < (uint32_t)kDecTile; i += kLebThreads) {
      const uint64_t p = b0 + i;
      if (p < a.nbytes && !(a.in[p] & 0x80)) ++c;
    }
  }
  c = wave_sum(c);
  if (lane_id() == 0) s_wave[wave_id()] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t t = 0;
    for (int w = 0; w < kLebWaves; ++w) t += s_wave[w];
    a.tile_terms[blockIdx.x] = t;
  }
}

// s_bytes[i] = in[b0 - kDecBack + i] (0 outside the stream).  Barrier.
__device__ __forceinline__ void dec_load_tile(const DecArgs& a, uint64_t b0, bool aligned,
                                              uint8_t* s_bytes) {
  if (threadIdx.x < kDecBack) {
    const int64_t p = (int64_t)b0 - kDecBack + threadIdx.x;
    s_bytes[threadIdx.x] = p >= 0 ? a.in[p] : 0;
  }
  if (aligned) {
    uint4* s4 = (uint4*)(s_bytes + kDecBack);
#pragma unroll
    for (int j = 0; j < kDecTile / 16 / kLebThreads; ++j) {
      const uint32_t q = j * kLebThreads + threadIdx.x;
      const uint64_t p = b0 + 16ull * q;
      s4[q] = p < a.nbytes ? load16(a.in, p, a.nbytes) : uint4{0u, 0u, 0u, 0u};
    }
  } else {
    for (uint32_t i = threadIdx.x; i < (uint32_t)kDecTile; i += kLebThreads) {
      const uint64_t p = b0 + i;
      s_bytes[kDecBack + i] = p < a.nbytes ? a.in[p] : 0;
    }
  }
  __syncthreads();
}

// Terminating bytes in this wavefront's 4 KiB of the tile (from LDS).
__device__ __forceinline__ uint32_t dec_wave_terms(const uint8_t* s_bytes, uint64_t b0,
                                                   uint64_t n) {
  const uint32_t* w32 = (const uint32_t*)(s_bytes + kDecBack) + wave_id() * (kDecWave / 4);
  const uint64_t pw = b0 + (uint64_t)wave_id() * kDecWave;
  uint32_t c = 0;
#pragma unroll 4
  for (int j = 0; j < kDecWave / 4 / 64; ++j) {
    const uint32_t q = j * 64 + lane_id();
    c += terms_in_word(w32[q], pw + 4ull * q, n);
  }
  return wave_sum(c);
}

// First entry id of this wavefront in the tile whose first is e0.
__device__ __forceinline__ uint64_t dec_wave_e0(uint64_t e0, const uint32_t* s_wterm) {
  uint64_t e = e0;
  for (uint32_t w = 0; w < wave_id(); ++w) e += s_wterm[w];
  return e;
}

// Every lane decodes 16 bytes per step: a wavefront covers 1 KiB per step
// and 4 KiB in kDecSteps steps.
constexpr int kDecSteps = kDecWave / (64 * 16);

// Byte j (0..15) of 16 bytes held as four dwords.
__device__ __forceinline__ uint32_t byte16(const leb_u32x4& v, int j) {
  return (v[j >> 2] >> (8 * (j & 3))) & 0xFFu;
}

// Bit j set: byte j ends a number (high bit clear).
__device__ __forceinline__ uint32_t ends16(const leb_u32x4& v) {
  uint32_t m = 0;
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    const uint32_t x = ~v[d] & 0x80808080u;
    m |= (((x >> 7) & 1u) | ((x >> 14) & 2u) | ((x >> 21) & 4u) | ((x >> 28) & 8u)) << (4 * d);
  }
  return m;
}

// The number that the bytes after the last terminating byte of the 16
// bytes P open (it continues past P): its payload so far and its length.
// Length 16 when P holds no terminating byte (a number over 10 bytes).
__device__ __forceinline__ void open_number(const leb_u32x4& P, uint64_t& v, uint32_t& len) {
  const uint32_t t = ends16(P);
  const int h = t ? 31 - __builtin_clz(t) : -1;
  len = (uint32_t)(15 - h);
  v = 0;
  // an open number of at most 9 bytes lies in bytes 7..15; a longer one is
  // malformed (decode16 flags it) and its value does not matter
#pragma unroll
  for (int j = 7; j < 16; ++j) {
    const int k = j - h - 1;   // byte k of the open number
    const bool in = k >= 0;
    const uint32_t sh = in ? 7u * (uint32_t)k : 0u;
    v |= in ? (uint64_t)(byte16(P, j) & 0x7Fu) << sh : 0ull;
  }
}

// Decodes the valid bytes (mask `valid`) of the 16 bytes C, continuing
// the open number (v_in, len_in): num[j] is the number that ends at byte j
// where bit j of the returned mask is set.  `bad`: a number over 10 bytes
// or over 64 bits.
__device__ __forceinline__ uint32_t decode16(const leb_u32x4& C, uint32_t valid, uint64_t v_in,
                                             uint32_t len_in, uint64_t* num, bool& bad) {
  const uint32_t ends = ends16(C) & valid;
  uint64_t acc = v_in;
  uint32_t k = len_in;
  bool b = false;
  // branch free: every byte is a few selects
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const uint32_t pl = byte16(C, j) & 0x7Fu;
    const bool vj = (valid >> j) & 1u;
    const uint32_t sh = k < 9 ? 7u * k : 63u;
    const uint64_t add = k <= 9 ? (uint64_t)(k < 9 ? pl : (pl & 1u)) << sh : 0ull;
    b |= vj & ((k == 9 && pl > 1) || k > 9);
    acc |= vj ? add : 0ull;
    k += vj ? 1u : 0u;
    num[j] = acc;
    const bool ej = (ends >> j) & 1u;
    acc = ej ? 0ull : acc;
    k = ej ? 0u : k;
  }
  bad |= b;
  return ends;
}

// Walks the segments of a tile's entries in increasing entry order.
struct SegCursor {
  uint32_t a;       // segment c.first + a (cached) or a (uncached)
  uint64_t lo;      // first entry of the segment
  uint64_t next;    // first entry of the next one (~0: none in this tile)
};

__device__ __forceinline__ SegCursor seg_cursor(const LebSegs& g, const TileSegs& c,
                                                const uint64_t* s_lo, uint64_t e) {
  SegCursor r{0, 0, ~0ull};
  if (g.num == 0) return r;
  if (c.cached) {
    const uint32_t n = c.last - c.first + 1;
    uint32_t a = 0, b = n;   // last a with s_lo[a] <= e
    while (b - a > 1) {
      const uint32_t mid = (a + b) >> 1;
      if (s_lo[mid] <= e) a = mid; else b = mid;
    }
    r.a = a;
    r.lo = s_lo[a];
    r.next = a + 1 < n ? s_lo[a + 1] : ~0ull;
  } else {
    r.a = seg_of(g, e);
    r.lo = g.offs[r.a];
    r.next = r.a + 1 < g.num ? g.offs[r.a + 1] : ~0ull;
  }
  return r;
}

// Moves the cursor to the segment of entry e (>= the cursor's entry) and
// returns whether e opens it, with the segment's base in `base`.
__device__ __forceinline__ bool seg_step(const LebSegs& g, const TileSegs& c,
                                         const uint64_t* s_lo, SegCursor& r, uint64_t e,
                                         int64_t& base) {
  if (g.num == 0) {
    base = seg_base0(g);
    return e == 0;
  }
  while (r.next <= e) {
    ++r.a;
    r.lo = r.next;
    if (c.cached) {
      r.next = r.a + 1 <= c.last - c.first ? s_lo[r.a + 1] : ~0ull;
    } else {
      r.next = r.a + 1 < g.num ? g.offs[r.a + 1] : ~0ull;
    }
  }
  const bool start = e == 0 || e == r.lo;
  base = start ? (int64_t)g.bases[c.cached ? c.first + r.a : r.a] : 0;
  return start;
}

// One step of one lane: the 16 bytes at tile offset q decoded, with the
// entry id of the lane's first number and the count.
struct LaneDec {
  uint64_t num[16];
  uint32_t ends;
  uint64_t e;        // entry id of the lane's first number
};

__device__ __forceinline__ void dec_lane_step(const DecArgs& a, const uint8_t* s_bytes,
                                              uint64_t b0, int it, uint64_t& e_step,
                                              LaneDec& d, bool& bad) {
  const uint32_t q = wave_id() * kDecWave + it * 1024 + lane_id() * 16;   // tile offset
  const uint64_t p = b0 + q;
  const leb_u32x4 C = *(const leb_u32x4*)(s_bytes + kDecBack + q);
  const leb_u32x4 P = *(const leb_u32x4*)(s_bytes + kDecBack + q - 16);
  uint32_t valid = 0;
  if (p < a.nbytes) valid = a.nbytes - p >= 16 ? 0xFFFFu : (1u << (a.nbytes - p)) - 1u;
  uint64_t v_in = 0;
  uint32_t len_in = 0;
  if (valid) open_number(P, v_in, len_in);
  d.ends = decode16(C, valid, v_in, len_in, d.num, bad);
  // the stream must not end inside a number
  if (valid && a.nbytes - p <= 16 && (s_bytes[kDecBack + q + (a.nbytes - p - 1)] & 0x80u))
    bad = true;
  const uint32_t cnt = __builtin_popcount(d.ends);
  const uint32_t incl = wave_incl_scan(cnt);
  d.e = e_step + incl - cnt;
  e_step += __shfl(incl, 63);
}

// Whether one of the lane's entries [d.e, d.e + count) opens a segment
// (`r` is the cursor at d.e).
__device__ __forceinline__ bool lane_opens(const LebSegs& g, const SegCursor& r,
                                           const LaneDec& d) {
  const uint64_t last = d.e + __builtin_popcount(d.ends) - 1;
  if (g.num == 0) return d.e == 0;
  return d.e == 0 || d.e == r.lo || r.next <= last;
}

// Segmented fold of one lane's numbers: whether one opens a segment, and
// the sum since the last that does (base + first term for it).
__device__ __forceinline__ void lane_fold(const DecArgs& a, const TileSegs& c,
                                          const uint64_t* s_lo, const LaneDec& d, uint32_t& f,
                                          uint64_t& v) {
  f = 0;
  v = 0;
  if (!d.ends) return;
  SegCursor r = seg_cursor(a.segs, c, s_lo, d.e);
  if (!lane_opens(a.segs, r, d)) {   // the common case: a plain sum
#pragma unroll
    for (int j = 0; j < 16; ++j) v += ((d.ends >> j) & 1u) ? d.num[j] : 0ull;
    return;
  }
  uint64_t e = d.e;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    if ((d.ends >> j) & 1u) {
      int64_t base;
      if (seg_step(a.segs, c, s_lo, r, e, base)) {
        f = 1;
        v = d.num[j] + (uint64_t)base;
      } else {
        v += d.num[j];
      }
      ++e;
    }
  }
}

// Segmented fold of this wavefront's entries (first entry id e): whether
// one opens a segment, and the sum since the last that does (or of all).
__device__ __forceinline__ void dec_wave_fold(const DecArgs& a, const TileSegs& c,
                                              const uint64_t* s_lo, const uint8_t* s_bytes,
                                              uint64_t b0, uint64_t e, bool& bad, uint32_t& f,
                                              uint64_t& v) {
  f = 0;
  v = 0;
  for (int it = 0; it < kDecSteps; ++it) {
    LaneDec d;
    dec_lane_step(a, s_bytes, b0, it, e, d, bad);
    uint32_t lf;
    uint64_t lv;
    lane_fold(a, c, s_lo, d, lf, lv);
    wave_seg_scan(lf, lv);
    const uint32_t sf = __shfl(lf, 63);
    const uint64_t sv = __shfl(lv, 63);
    if (sf) {
      f = 1;
      v = sv;
    } else {
      v += sv;
    }
  }
}

// First entry and segment range of every byte tile, after the count scan:
// one wavefront per group of 64 tiles (a tile per lane, an exclusive scan
// of their terms), so that the decode kernels take them with one load
// instead of a group sum and a search per workgroup.
__global__ __launch_bounds__(256) void dec_recs_kernel(DecArgs a, uint64_t btiles) {
  const uint64_t g = (uint64_t)blockIdx.x * 4 + wave_id();
  const uint64_t t = g * kTilesPerGroup + lane_id();
  if (g * kTilesPerGroup >= btiles) return;   // uniform per wavefront
  const uint32_t terms = t < btiles ? a.tile_terms[t] : 0u;
  const uint32_t incl = wave_incl_scan(terms);
  if (t >= btiles) return;
  DecTileRec r{a.group_excl[g] + (incl - terms), 0u, 0u, 0ull};
  if (terms && a.segs.num) {
    r.first = seg_of(a.segs, r.e0);
    r.last = seg_of(a.segs, r.e0 + terms - 1);
    r.lo0 = a.segs.offs[r.first];
  }
  a.tile_recs[t] = r;
}

// The tile's segments from its record; their starts go to s_lo, which the
// caller's next barrier publishes.
__device__ __forceinline__ TileSegs dec_tile_segs(const DecArgs& a, const DecTileRec& r,
                                                  uint64_t* s_lo) {
  TileSegs c{0, 0, false, 0};
  if (a.segs.num == 0) return c;
  c.first = r.first;
  c.last = r.last;
  c.lo0 = r.lo0;
  const uint32_t n = c.last - c.first + 1;
  if (n <= (uint32_t)kSegLds) {
    for (uint32_t j = threadIdx.x; j < n; j += kLebThreads)
      s_lo[j] = j == 0 ? r.lo0 : a.segs.offs[c.first + j];
    c.cached = true;
  }
  return c;
}

__global__ __launch_bounds__(kLebThreads) void dec_fold_kernel(DecArgs a, bool aligned) {
  __shared__ __align__(16) uint8_t s_bytes[kDecBack + kDecTile];
  __shared__ uint64_t s_lo[kSegLds];
  __shared__ uint32_t s_wterm[kLebWaves];
  __shared__ uint32_t s_wf[kLebWaves];
  __shared__ uint64_t s_wv[kLebWaves];
  const uint64_t tile = blockIdx.x;
  const uint64_t b0 = tile * kDecTile;
  const DecTileRec rec = a.tile_recs[tile];
  dec_load_tile(a, b0, aligned, s_bytes);                                    // barrier
  const uint64_t e0 = rec.e0;
  const uint32_t terms = a.tile_terms[tile];
  const uint32_t wt = dec_wave_terms(s_bytes, b0, a.nbytes);
  if (lane_id() == 0) s_wterm[wave_id()] = wt;
  const TileSegs c = dec_tile_segs(a, rec, s_lo);
  __syncthreads();
  bool bad = false;
  if (terms == 0) {   // uniform: no number ends in this tile
    if (threadIdx.x == 0) {
      a.tile_f[tile] = 0;
      a.tile_v[tile] = 0;
    }
    const uint64_t last = a.nbytes - 1;   // the stream must not end inside a number
    if (threadIdx.x == 0 && last >= b0 && last < b0 + kDecTile &&
        (s_bytes[kDecBack + (last - b0)] & 0x80))
      bad = true;
    if (bad) raise_flag(a.err);
    return;
  }
  uint32_t f;
  uint64_t v;
  dec_wave_fold(a, c, s_lo, s_bytes, b0, dec_wave_e0(e0, s_wterm), bad, f, v);
  if (lane_id() == 0) {
    s_wf[wave_id()] = f;
    s_wv[wave_id()] = v;
    a.wave_f[tile * kLebWaves + wave_id()] = f;   // read back by dec_write
    a.wave_v[tile * kLebWaves + wave_id()] = v;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t tf = 0;
    uint64_t tv = 0;
    for (int w = 0; w < kLebWaves; ++w) {
      if (s_wf[w]) {
        tf = 1;
        tv = s_wv[w];
      } else {
        tv += s_wv[w];
      }
    }
    a.tile_f[tile] = tf;
    a.tile_v[tile] = tv;
  }
  if (bad) raise_flag(a.err);
}

// Segmented fold of tiles [lo, end) (end - lo <= 64) by one wavefront.
__device__ __forceinline__ void seg_fold_tiles(const uint32_t* f, const uint64_t* v, uint64_t lo,
                                               uint64_t end, uint32_t& out_f, uint64_t& out_v) {
  const uint64_t t = lo + lane_id();
  const bool in = t < end;
  const uint32_t tf = in ? f[t] : 0;
  const uint64_t tv = in ? v[t] : 0;
  const uint64_t fm = __ballot(tf != 0);
  uint64_t x = tv;
  if (fm) {
    const uint32_t L = 63 - __builtin_clzll(fm);
    x = lane_id() >= L ? tv : 0;
  }
  out_f = fm != 0;
  out_v = wave_sum(x);
}

__global__ __launch_bounds__(64) void seg_group_sum_kernel(const uint32_t* tile_f,
                                                           const uint64_t* tile_v,
                                                           uint64_t num_tiles, uint32_t* gsum_f,
                                                           uint64_t* gsum_v) {
  const uint64_t lo = (uint64_t)blockIdx.x * kTilesPerGroup;
  const uint64_t end = lo + kTilesPerGroup < num_tiles ? lo + kTilesPerGroup : num_tiles;
  uint32_t f;
  uint64_t v;
  seg_fold_tiles(tile_f, tile_v, lo, end, f, v);
  if (lane_id() == 0) {
    gsum_f[blockIdx.x] = f;
    gsum_v[blockIdx.x] = v;
  }
}

// Exclusive segmented scan of the group folds: gexcl_v[g] = the index of
// the last entry before group g (one workgroup, passes of 1024 groups).
// Without flags (gsum_f NULL) it is a plain exclusive scan; d_total
// (nullable) gets the inclusive value at the end.
constexpr int kSegScanThreads = 1024;
__global__ __launch_bounds__(kSegScanThreads) void seg_group_scan_kernel(const uint32_t* gsum_f,
                                                                         const uint64_t* gsum_v,
                                                                         uint64_t num_groups,
                                                                         uint64_t* gexcl_v,
                                                                         uint64_t* d_total) {
  __shared__ uint32_t s_f[kSegScanThreads / 64];
  __shared__ uint64_t s_v[kSegScanThreads / 64];
  __shared__ uint64_t s_carry;
  const uint32_t lane = lane_id(), wave = threadIdx.x >> 6;
  if (threadIdx.x == 0) s_carry = 0;
  __syncthreads();
  for (uint64_t base = 0; base < num_groups; base += kSegScanThreads) {
    const uint64_t i = base + threadIdx.x;
    uint32_t f = (gsum_f && i < num_groups) ? gsum_f[i] : 0;
    uint64_t v = i < num_groups ? gsum_v[i] : 0;
    wave_seg_scan(f, v);
    if (lane == 63) {
      s_f[wave] = f;
      s_v[wave] = v;
    }
    __syncthreads();
    uint64_t before = s_carry;   // index of the entry before this wavefront's groups
    for (uint32_t w = 0; w < wave; ++w) before = s_f[w] ? s_v[w] : before + s_v[w];
    const uint64_t incl = f ? v : before + v;
    const uint64_t prev = __shfl_up(incl, 1);
    if (i < num_groups) gexcl_v[i] = lane == 0 ? before : prev;
    __syncthreads();
    if (threadIdx.x == kSegScanThreads - 1) s_carry = incl;
    __syncthreads();
  }
  if (d_total && threadIdx.x == 0) *d_total = s_carry;
}

// Entries one wavefront decodes in one step, at most (64 lanes x 16 bytes).
constexpr int kDecStepEntries = 64 * 16;

__global__ __launch_bounds__(kLebThreads) void dec_write_kernel(DecArgs a, bool aligned) {
  __shared__ __align__(16) uint8_t s_bytes[kDecBack + kDecTile];
  __shared__ uint64_t s_lo[kSegLds];
  __shared__ uint32_t s_wterm[kLebWaves];
  __shared__ uint64_t s_carry;
  // every wavefront's decoded indices of one step, written out coalesced
  __shared__ uint64_t s_out[kLebWaves][kDecStepEntries];
  const uint64_t tile = blockIdx.x;
  const uint32_t terms = a.tile_terms[tile];
  if (terms == 0) return;   // uniform
  const uint64_t b0 = tile * kDecTile;
  const DecTileRec rec = a.tile_recs[tile];
  dec_load_tile(a, b0, aligned, s_bytes);                                    // barrier
  const uint64_t e0 = rec.e0;
  if (e0 >= a.capacity) return;   // uniform: nothing of this tile is kept
  const uint32_t lane = lane_id(), wave = wave_id();
  if (threadIdx.x < 64) {   // index of the entry just before the tile
    const uint64_t g = tile / kTilesPerGroup;
    uint32_t f;
    uint64_t v;
    seg_fold_tiles(a.tile_f, a.tile_v, g * kTilesPerGroup, tile, f, v);
    if (threadIdx.x == 0) s_carry = f ? v : a.gexcl_v[g] + v;
  }
  const uint32_t wt = dec_wave_terms(s_bytes, b0, a.nbytes);
  if (lane == 0) s_wterm[wave] = wt;
  const TileSegs c = dec_tile_segs(a, rec, s_lo);
  __syncthreads();
  const uint64_t ew = dec_wave_e0(e0, s_wterm);
  // index of the entry before this wavefront's first, from dec_fold's
  // per-wavefront folds
  uint64_t run = s_carry;
  for (uint32_t w = 0; w < wave; ++w)
    run = a.wave_f[tile * kLebWaves + w] ? a.wave_v[tile * kLebWaves + w]
                                         : run + a.wave_v[tile * kLebWaves + w];
  bool bad = false;   // reported by dec_fold
  uint64_t* so = s_out[wave];
  uint64_t e = ew;
  for (int it = 0; it < kDecSteps; ++it) {
    const uint64_t e_step = e;
    LaneDec d;
    dec_lane_step(a, s_bytes, b0, it, e, d, bad);
    uint32_t lf;
    uint64_t lv;
    lane_fold(a, c, s_lo, d, lf, lv);
    // index before this lane's first number: segmented exclusive scan
    uint32_t sf = lf;
    uint64_t sv = lv;
    wave_seg_scan(sf, sv);
    uint32_t xf = __shfl_up(sf, 1);
    uint64_t xv = __shfl_up(sv, 1);
    if (lane == 0) {
      xf = 0;
      xv = 0;
    }
    uint64_t y = xf ? xv : run + xv;
    const uint32_t f63 = __shfl(sf, 63);
    const uint64_t v63 = __shfl(sv, 63);
    run = f63 ? v63 : run + v63;
    if (d.ends) {
      SegCursor r = seg_cursor(a.segs, c, s_lo, d.e);
      uint64_t k = d.e;
      if (!lane_opens(a.segs, r, d)) {   // the common case: running sums
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          if ((d.ends >> j) & 1u) {
            y += d.num[j];
            so[k - e_step] = y;
            ++k;
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          if ((d.ends >> j) & 1u) {
            int64_t base;
            y = seg_step(a.segs, c, s_lo, r, k, base) ? d.num[j] + (uint64_t)base : y + d.num[j];
            so[k - e_step] = y;
            ++k;
          }
        }
      }
    }
    // the wavefront's entries of this step are contiguous: store them
    // coalesced from LDS (LDS operations of one wavefront complete in order)
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const uint32_t n = (uint32_t)(e - e_step);
    for (uint32_t i = lane; i < n; i += 64) {
      const uint64_t k = e_step + i;
      if (k < a.capacity) a.out[k] = (int64_t)so[i];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();   // so[] is rewritten by the next step
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

// Global index -> tensor holding it (tbases[t] <= y < tbases[t + 1]).
__device__ __forceinline__ uint32_t dec_find_tensor(const uint64_t* tbases, uint32_t T,
                                                    uint64_t y) {
  uint32_t lo = 0, hi = T;
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) >> 1;
    if (tbases[mid] <= y) lo = mid; else hi = mid;
  }
  return lo;
}

// Decode-in-apply: decodes like dec_write_kernel, but every number's
// index y receives its entry's word, w[y] = val[k] in the tensor holding
// y, with no index stream written.  Each step's indices are staged in LDS
// so that, as in the plain apply, every store instruction covers 64
// consecutive entries and the words are loaded coalesced.  Entries past
// the value count, indices outside the tensor list, and a stream whose
// entry count differs from the value count raise the error flag; those
// words are left alone.
__global__ __launch_bounds__(kLebThreads) void dec_apply_kernel(DecArgs a, bool aligned) {
  __shared__ __align__(16) uint8_t s_bytes[kDecBack + kDecTile];
  __shared__ uint64_t s_lo[kSegLds];
  __shared__ uint32_t s_wterm[kLebWaves];
  __shared__ uint64_t s_carry;
  __shared__ uint64_t s_out[kLebWaves][kDecStepEntries];
  const uint64_t tile = blockIdx.x;
  if (tile == 0 && threadIdx.x == 0 && *a.d_count != a.capacity) raise_flag(a.err);
  const uint32_t terms = a.tile_terms[tile];
  if (terms == 0) return;   // uniform
  const uint64_t b0 = tile * kDecTile;
  const DecTileRec rec = a.tile_recs[tile];
  dec_load_tile(a, b0, aligned, s_bytes);                                    // barrier
  const uint64_t e0 = rec.e0;
  if (e0 >= a.capacity) {   // uniform: no value for any entry of this tile
    if (threadIdx.x == 0) raise_flag(a.err);
    return;
  }
  const uint32_t lane = lane_id(), wave = wave_id();
  if (threadIdx.x < 64) {   // index of the entry just before the tile
    const uint64_t g = tile / kTilesPerGroup;
    uint32_t f;
    uint64_t v;
    seg_fold_tiles(a.tile_f, a.tile_v, g * kTilesPerGroup, tile, f, v);
    if (threadIdx.x == 0) s_carry = f ? v : a.gexcl_v[g] + v;
  }
  const uint32_t wt = dec_wave_terms(s_bytes, b0, a.nbytes);
  if (lane == 0) s_wterm[wave] = wt;
  const TileSegs c = dec_tile_segs(a, rec, s_lo);
  __syncthreads();
  const uint64_t ew = dec_wave_e0(e0, s_wterm);
  uint64_t run = s_carry;
  for (uint32_t w = 0; w < wave; ++w)
    run = a.wave_f[tile * kLebWaves + w] ? a.wave_v[tile * kLebWaves + w]
                                         : run + a.wave_v[tile * kLebWaves + w];
  const uint64_t total = a.tbases[a.num_tensors];
  bool bad = false;
  uint32_t t = 0;                 // the tensor [lo, hi) last written by this lane
  uint64_t lo = 1, hi = 0;
  uint16_t* base_ptr = nullptr;
  uint64_t* so = s_out[wave];
  uint64_t e = ew;
  for (int it = 0; it < kDecSteps; ++it) {
    const uint64_t e_step = e;
    LaneDec d;
    dec_lane_step(a, s_bytes, b0, it, e, d, bad);
    uint32_t lf;
    uint64_t lv;
    lane_fold(a, c, s_lo, d, lf, lv);
    uint32_t sf = lf;
    uint64_t sv = lv;
    wave_seg_scan(sf, sv);
    uint32_t xf = __shfl_up(sf, 1);
    uint64_t xv = __shfl_up(sv, 1);
    if (lane == 0) {
      xf = 0;
      xv = 0;
    }
    uint64_t y = xf ? xv : run + xv;
    const uint32_t f63 = __shfl(sf, 63);
    const uint64_t v63 = __shfl(sv, 63);
    run = f63 ? v63 : run + v63;
    if (d.ends) {
      SegCursor r = seg_cursor(a.segs, c, s_lo, d.e);
      uint64_t k = d.e;
      if (!lane_opens(a.segs, r, d)) {   // the common case: running sums
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          if ((d.ends >> j) & 1u) {
            y += d.num[j];
            so[k - e_step] = y;
            ++k;
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          if ((d.ends >> j) & 1u) {
            int64_t base;
            y = seg_step(a.segs, c, s_lo, r, k, base) ? d.num[j] + (uint64_t)base : y + d.num[j];
            so[k - e_step] = y;
            ++k;
          }
        }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const uint32_t n = (uint32_t)(e - e_step);
    for (uint32_t i = lane; i < n; i += 64) {
      const uint64_t k = e_step + i;
      const uint64_t yi = so[i];
      if (k < a.capacity && yi < total) {
        if (!(yi >= lo && yi < hi)) {
          t = dec_find_tensor(a.tbases, a.num_tensors, yi);
          lo = a.tbases[t];
          hi = a.tbases[t + 1];
          base_ptr = a.ptrs[t];
        }
        __builtin_nontemporal_store(a.val[k], base_ptr + (yi - lo));
      } else {
        bad = true;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();   // so[] is rewritten by the next step
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  if (bad) raise_flag(a.err);
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
  L.tile_segs = align_up(L.group_excl + 8 * groups);
  L.stage = align_up(L.tile_segs + sizeof(EncTileSegs) * tiles);
  L.total = align_up(L.stage + (size_t)kEncSlot * tiles);
  return L;
}

DecLayout dec_layout(uint64_t nbytes) {
  DecLayout L;
  const uint64_t bt = dec_tiles(nbytes), gb = groups_for(bt);
  L.btiles = bt;
  L.tile_terms = 0;
  L.group_sum = align_up(4 * bt);
  L.group_excl = align_up(L.group_sum + 8 * gb);
  L.tile_f = align_up(L.group_excl + 8 * gb);
  L.tile_v = align_up(L.tile_f + 4 * bt);
  L.wave_f = align_up(L.tile_v + 8 * bt);
  L.wave_v = align_up(L.wave_f + 4 * kLebWaves * bt);
  L.gsum_f = align_up(L.wave_v + 8 * kLebWaves * bt);
  L.gsum_v = align_up(L.gsum_f + 4 * gb);
  L.gexcl_v = align_up(L.gsum_v + 8 * gb);
  L.tile_recs = align_up(L.gexcl_v + 8 * gb);
  L.total = align_up(L.tile_recs + sizeof(DecTileRec) * bt);
  return L;
}

uint32_t enc_grid(uint64_t count, bool count_on_device) {
  const uint64_t tiles = enc_tiles(count);
  const uint64_t cap = count_on_device ? 2048 : 0xFFFFFFFFull;
  return (uint32_t)(tiles < cap ? (tiles ? tiles : 1) : cap);
}

hipError_t launch_leb128_encode(EncArgs a, char* ws, const EncLayout& L, hipStream_t stream) {
  const uint64_t tiles = enc_tiles(a.count);   // at most
  a.tile_bytes = (uint32_t*)(ws + L.tile_bytes);
  a.group_excl = (uint64_t*)(ws + L.group_excl);
  a.stage = (uint8_t*)(ws + L.stage);
  a.tile_segs = (EncTileSegs*)(ws + L.tile_segs);
  hipError_t e;
  if (tiles == 0) {
    e = launch_reset(a.d_nbytes, nullptr, 0, stream);
  } else {
    const uint32_t grid = enc_grid(a.count, a.d_count_in != nullptr);
    const uint64_t groups = groups_for(tiles);
    e = hipSuccess;
    if (a.segs.num) {
      const uint64_t blocks = (tiles + 255) / 256;
      hipLaunchKernelGGL(enc_segs_kernel, dim3((uint32_t)(blocks < 2048 ? blocks : 2048)),
                         dim3(256), 0, stream, a);
      e = hipGetLastError();
    }
    if (e == hipSuccess) {
      hipLaunchKernelGGL(enc_stage_kernel, dim3(grid), dim3(kLebThreads), 0, stream, a);
      e = hipGetLastError();
    }
    if (e == hipSuccess) {
      hipLaunchKernelGGL(enc_group_sum_kernel, dim3((uint32_t)groups), dim3(64), 0, stream, a,
                         (uint64_t*)(ws + L.group_sum));
      e = hipGetLastError();
    }
    if (e == hipSuccess) {
      hipLaunchKernelGGL(seg_group_scan_kernel, dim3(1), dim3(kSegScanThreads), 0, stream,
                         (const uint32_t*)nullptr, (const uint64_t*)(ws + L.group_sum), groups,
                         a.group_excl, a.d_nbytes);
      e = hipGetLastError();
    }
    if (e == hipSuccess) {
      hipLaunchKernelGGL(enc_copy_kernel, dim3(grid), dim3(kLebThreads), 0, stream, a);
      e = hipGetLastError();
    }
  }
  if (e == hipSuccess && a.seg_byte_offsets) {
    const uint32_t n = a.segs.num + 1;
    hipLaunchKernelGGL(enc_seg_fix_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, a);
    e = hipGetLastError();
  }
  return e;
}

// The decoder's single segment (num == 0) is based at 0.
hipError_t launch_leb128_decode(DecArgs a, const DecLayout& L, char* ws, hipStream_t stream,
                                bool apply) {
  hipError_t e;
  if (L.btiles == 0) return launch_reset(a.d_count, nullptr, 0, stream);
  a.segs.base0 = 0;
  a.tile_terms = (uint32_t*)(ws + L.tile_terms);
  a.group_excl = (uint64_t*)(ws + L.group_excl);
  a.tile_f = (uint32_t*)(ws + L.tile_f);
  a.tile_v = (uint64_t*)(ws + L.tile_v);
  a.wave_f = (uint32_t*)(ws + L.wave_f);
  a.wave_v = (uint64_t*)(ws + L.wave_v);
  a.gexcl_v = (uint64_t*)(ws + L.gexcl_v);
  const bool aligned = ((uintptr_t)a.in & 15u) == 0;
  const dim3 grid((uint32_t)L.btiles), block(kLebThreads);
  hipLaunchKernelGGL(dec_count_kernel, grid, block, 0, stream, a, aligned);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if ((e = launch_group_scan(a.tile_terms, L.btiles, (uint64_t*)(ws + L.group_sum), a.group_excl,
                             a.d_count, stream)) != hipSuccess)
    return e;
  a.tile_recs = (DecTileRec*)(ws + L.tile_recs);
  const uint64_t rec_blocks = (groups_for(L.btiles) + 3) / 4;
  hipLaunchKernelGGL(dec_recs_kernel, dim3((uint32_t)rec_blocks), dim3(256), 0, stream, a,
                     L.btiles);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(dec_fold_kernel, grid, block, 0, stream, a, aligned);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const uint64_t groups = groups_for(L.btiles);
  hipLaunchKernelGGL(seg_group_sum_kernel, dim3((uint32_t)groups), dim3(64), 0, stream, a.tile_f,
                     a.tile_v, L.btiles, (uint32_t*)(ws + L.gsum_f), (uint64_t*)(ws + L.gsum_v));
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(seg_group_scan_kernel, dim3(1), dim3(kSegScanThreads), 0, stream,
                     (const uint32_t*)(ws + L.gsum_f), (const uint64_t*)(ws + L.gsum_v), groups,
                     a.gexcl_v, (uint64_t*)nullptr);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (apply)
    hipLaunchKernelGGL(dec_apply_kernel, grid, block, 0, stream, a, aligned);
  else
    hipLaunchKernelGGL(dec_write_kernel, grid, block, 0, stream, a, aligned);
  return hipGetLastError();
}

}  // namespace aurora
