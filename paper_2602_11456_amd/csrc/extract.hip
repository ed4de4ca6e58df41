// Sparse delta extraction on gfx950: one pass over both bf16 copies that
// keeps every word whose bits changed and writes the kept positions and new
// words, in ascending position order, as two dense streams (AuroraRL
// Sec. 5.1, "Sparse encoding").
//
// Per workgroup (one tile of 8192 words, tile id = workgroup id):
//   1. find the tile's tensor slice (tile -> slice map for tensor lists);
//   2. read 16 bytes of each copy per lane per unrolled step;
//   3. compare 16-bit words, count changes per lane, turn the counts into
//      lane prefixes with four ballots + mbcnt (bit-sliced prefix sum);
//   4. combine wavefront totals through LDS into the tile's aggregate;
//   5. decoupled look-back over the tile-state array (Merrill & Garland,
//      "Single-pass Parallel Prefix Scan with Decoupled Look-back", 2016)
//      to learn how many kept words precede the tile;
//   6. write the kept (index, word) pairs at their final positions.
//
// Forward progress does not rest on the order in which workgroups are
// dispatched: a look-back that has waited `spin_limit` polls for a
// predecessor that has published nothing counts that predecessor's tile
// itself (one wavefront reads its 8192 words) and goes on.  A tile id
// counter would also guarantee progress, but one device-scope atomic per
// tile on a single address serialises the whole grid at the memory side.
#include "delta_internal.h"

namespace aurora {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint64_t load_state(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_state(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

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

// Loads group g (words 8g - head .. 8g - head + 7 of the slice).  Words
// outside [0, n) read as equal zeros, so they never count as changed.
__device__ __forceinline__ void load_group(const TensorDesc& d, int64_t g,
                                           u32x4& p, u32x4& q) {
  const int64_t e0 = 8 * g - (int64_t)d.head;
  if (d.vec && e0 >= 0 && e0 + 8 <= (int64_t)d.n) {
    const u32x4* pp = reinterpret_cast<const u32x4*>(
        reinterpret_cast<uintptr_t>(d.prev) - 2u * d.head) + g;
    const u32x4* qq = reinterpret_cast<const u32x4*>(
        reinterpret_cast<uintptr_t>(d.next) - 2u * d.head) + g;
    p = __builtin_nontemporal_load(pp);
    q = __builtin_nontemporal_load(qq);
  } else {
    uint32_t pw[4] = {0, 0, 0, 0}, qw[4] = {0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int64_t e = e0 + j;
      if (e >= 0 && e < (int64_t)d.n) {
        pw[j >> 1] |= (uint32_t)d.prev[e] << (16 * (j & 1));
        qw[j >> 1] |= (uint32_t)d.next[e] << (16 * (j & 1));
      }
    }
    p = u32x4{pw[0], pw[1], pw[2], pw[3]};
    q = u32x4{qw[0], qw[1], qw[2], qw[3]};
  }
}

// Bit j of the result is set when word j of the group changed.
__device__ __forceinline__ uint32_t changed_mask(const u32x4& p, const u32x4& q) {
  uint32_t m = 0;
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    const uint32_t x = p[d] ^ q[d];
    m |= (uint32_t)((x & 0xFFFFu) != 0) << (2 * d);
    m |= (uint32_t)((x >> 16) != 0) << (2 * d + 1);
  }
  return m;
}

__device__ __forceinline__ uint32_t wave_sum32(uint32_t v) {
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) v += __shfl_xor(v, s);
  return v;
}

template <bool kMulti>
__device__ __forceinline__ TensorDesc tile_desc(const ExtractArgs& a, uint64_t tile) {
  return kMulti ? a.table[a.tile_map[tile]] : a.single;
}

// Changed words of tile t, counted by one wavefront (look-back fallback).
// A cold path: plain 2-byte loads keep its register footprint small.
template <bool kMulti>
__device__ __forceinline__ uint32_t count_tile_wave(const ExtractArgs& a, uint64_t t, uint32_t lane) {
  const TensorDesc d = tile_desc<kMulti>(a, t);
  const int64_t e0 = (int64_t)((t - d.first_tile) * kElemsPerTile) - (int64_t)d.head;
  uint32_t c = 0;
#pragma unroll 1
  for (int64_t i = lane; i < kElemsPerTile; i += 64) {
    const int64_t e = e0 + i;
    if (e >= 0 && e < (int64_t)d.n) c += (d.prev[e] != d.next[e]) ? 1u : 0u;
  }
  return wave_sum32(c);
}

// Per-lane state of one tile after the compare: which words changed and
// where they go inside the tile's output run.
struct TileScan {
  u32x4 q[kChunks];               // new words
  uint32_t mask[kChunks];         // bit j: word j of the lane's group changed
  uint32_t lane_prefix[kChunks];  // kept words of lower lanes in the same chunk
  uint32_t chunk_base[kChunks];   // wave-uniform: kept words of earlier chunks
  uint32_t wave_total;
};

__device__ __forceinline__ void scan_tile(const TensorDesc& d, int64_t g0, TileScan& s) {
  u32x4 p[kChunks];
#pragma unroll
  for (int u = 0; u < kChunks; ++u) load_group(d, g0 + 64 * u, p[u], s.q[u]);
  s.wave_total = 0;
#pragma unroll
  for (int u = 0; u < kChunks; ++u) {
    s.mask[u] = changed_mask(p[u], s.q[u]);
    // bit-sliced prefix sum of the per-lane counts (0..8) over the wavefront
    const uint32_t c = __popc(s.mask[u]);
    const uint64_t b0 = __ballot(c & 1), b1 = __ballot(c & 2);
    const uint64_t b2 = __ballot(c & 4), b3 = __ballot(c & 8);
    s.lane_prefix[u] = mbcnt64(b0) + 2 * mbcnt64(b1) + 4 * mbcnt64(b2) + 8 * mbcnt64(b3);
    s.chunk_base[u] = s.wave_total;
    s.wave_total += __popcll(b0) + 2 * __popcll(b1) + 4 * __popcll(b2) + 8 * __popcll(b3);
  }
}

__device__ __forceinline__ uint16_t word_of(const u32x4& q, int j) {
  const uint32_t dw = q[j >> 1];
  return (uint16_t)((j & 1) ? (dw >> 16) : (dw & 0xFFFFu));
}

template <typename IdxT, bool kMulti>
__global__ __launch_bounds__(kThreads) void extract_kernel(ExtractArgs a) {
  __shared__ uint32_t s_wave_total[kWaves];
  __shared__ uint64_t s_tile_excl;
  // kept entries of the tile in output order: (new word << 16) | word offset in tile
  __shared__ uint32_t s_stage[kStageCap];

  const uint64_t tile = blockIdx.x;
  const TensorDesc d = tile_desc<kMulti>(a, tile);
  const uint64_t local_tile = tile - d.first_tile;
  const uint32_t lane = lane_id();
  const uint32_t wave = threadIdx.x >> 6;
  const uint32_t lane_group = wave * kGroupsPerWave + lane;   // group of chunk 0 in the tile
  const int64_t g0 = (int64_t)(local_tile * kGroupsPerTile) + lane_group;
  // slice word index of the tile's word 0 (negative inside a misaligned head)
  const int64_t tile_e0 = (int64_t)(local_tile * kElemsPerTile) - (int64_t)d.head;

  uint32_t wave_excl = 0, tile_total = 0;
  {
    TileScan s;
    scan_tile(d, g0, s);
    if (lane == 0) s_wave_total[wave] = s.wave_total;
    __syncthreads();
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const uint32_t t = s_wave_total[w];
      wave_excl += (w < (int)wave) ? t : 0u;
      tile_total += t;
    }
    // Stage the kept entries in LDS now, so nothing of the tile stays live
    // in registers through the look-back; the global writes after it are
    // then contiguous runs.
    if (tile_total <= (uint32_t)kStageCap) {
#pragma unroll
      for (int u = 0; u < kChunks; ++u) {
        uint32_t m = s.mask[u];
        uint32_t r = wave_excl + s.chunk_base[u] + s.lane_prefix[u];
        const uint32_t w0 = (lane_group + 64 * u) * 8;
        while (m) {
          const int j = __builtin_ctz(m);
          m &= m - 1;
          s_stage[r++] = ((uint32_t)word_of(s.q[u], j) << 16) | (w0 + j);
        }
      }
    }
  }

  // Decoupled look-back, done by wavefront 0.
  if (wave == 0) {
    uint64_t excl = 0;
    if (tile == 0) {
      if (lane == 0) store_state(&a.states[0], kStatePrefix | tile_total);
    } else {
      if (lane == 0) store_state(&a.states[tile], kStateAggregate | tile_total);
      int64_t top = (int64_t)tile - 1;
      for (;;) {
        const int64_t t = top - (int64_t)lane;
        uint64_t st = (t >= 0) ? load_state(&a.states[t]) : kStatePrefix;
        uint64_t need, prefix_lanes;
        uint32_t spins = 0;
        for (;;) {
          const uint64_t empty = __ballot((st & kStateFlagMask) == kStateEmpty);
          prefix_lanes = __ballot((st & kStateFlagMask) == kStatePrefix);
          // lanes that count: up to and including the nearest full prefix
          need = prefix_lanes ? (((prefix_lanes & (0 - prefix_lanes)) << 1) - 1) : ~0ull;
          const uint64_t pending = empty & need;
          if (pending == 0) break;
          if (spins >= a.spin_limit) {
            // count the nearest silent predecessor ourselves
            const uint32_t l = (uint32_t)__builtin_ctzll(pending);
            const uint32_t agg = count_tile_wave<kMulti>(a, (uint64_t)(top - (int64_t)l), lane);
            if (lane == l) st = kStateAggregate | agg;
            if (lane == 0)
              __hip_atomic_fetch_add(&a.ctrl->fallbacks, 1u, __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT);
            spins = 0;
            continue;
          }
          ++spins;
          __builtin_amdgcn_s_sleep(1);
          if ((pending >> lane) & 1ull) st = load_state(&a.states[t]);
        }
        const uint64_t v = ((need >> lane) & 1ull) ? (st & kStateValueMask) : 0ull;
        excl += wave_sum64(v);
        if (prefix_lanes) break;
        top -= 64;
      }
      if (lane == 0) store_state(&a.states[tile], kStatePrefix | (excl + tile_total));
    }
    if (lane == 0) s_tile_excl = excl;
  }
  __syncthreads();
  const uint64_t tile_excl = s_tile_excl;

  if (threadIdx.x == 0) {
    // tensor_offsets: the first tile of a slice owns the slots of its own
    // tensor and of the empty tensors just before it; the last tile owns
    // the slots after its tensor (trailing empty tensors and the total).
    if (a.d_tensor_offsets && local_tile == 0) {
      for (uint32_t s = d.off_lo; s <= d.slot; ++s) a.d_tensor_offsets[s] = tile_excl;
    }
    if (tile == a.num_tiles - 1) {
      const uint64_t total = tile_excl + tile_total;
      *a.d_count = total;
      if (a.d_tensor_offsets) {
        for (uint32_t s = d.slot + 1; s <= a.num_tensors; ++s) a.d_tensor_offsets[s] = total;
      }
    }
  }

  IdxT* out_idx = reinterpret_cast<IdxT*>(a.out_idx);
  const int64_t out_base = (int64_t)d.base + tile_e0;
  if (tile_total <= (uint32_t)kStageCap) {
    // contiguous run [tile_excl, tile_excl + tile_total) of the output
    for (uint32_t r = threadIdx.x; r < tile_total; r += kThreads) {
      const uint64_t pos = tile_excl + r;
      if (pos < a.capacity) {
        const uint32_t e = s_stage[r];
        out_idx[pos] = (IdxT)(out_base + (e & 0xFFFFu));
        a.out_val[pos] = (uint16_t)(e >> 16);
      }
    }
  } else {
    // more kept words than the stage holds: read the tile again and write
    // each entry from registers
    TileScan s;
    scan_tile(d, g0, s);
#pragma unroll
    for (int u = 0; u < kChunks; ++u) {
      uint32_t m = s.mask[u];
      uint64_t pos = tile_excl + wave_excl + s.chunk_base[u] + s.lane_prefix[u];
      const int64_t e0 = out_base + (int64_t)(lane_group + 64 * u) * 8;
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
}

__global__ void reset_kernel(Control* ctrl, uint64_t* states, uint64_t num_tiles,
                             uint64_t* d_count, uint64_t* d_offsets, uint32_t num_offsets) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  const uint64_t i0 = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (uint64_t i = i0; i < num_tiles; i += stride) states[i] = kStateEmpty;
  if (d_offsets)
    for (uint64_t i = i0; i < num_offsets; i += stride) d_offsets[i] = 0;
  if (i0 == 0) {
    ctrl->fallbacks = 0;
    *d_count = 0;
  }
}

__global__ void upload_words_kernel(WordBatch b, uint64_t* dst) {
  for (uint32_t i = threadIdx.x; i < b.count; i += blockDim.x) dst[i] = b.w[i];
}

__global__ void build_tile_map_kernel(const TensorDesc* table, uint32_t* tile_map) {
  const uint32_t t = blockIdx.x;
  const TensorDesc d = table[t];
  const uint64_t nt = tiles_for(d.n, d.head);
  for (uint64_t i = threadIdx.x; i < nt; i += blockDim.x) tile_map[d.first_tile + i] = t;
}

hipError_t launch_reset(Control* ctrl, uint64_t* states, uint64_t num_tiles,
                        uint64_t* d_count, uint64_t* d_offsets, uint32_t num_offsets,
                        hipStream_t stream) {
  uint64_t work = num_tiles > num_offsets ? num_tiles : num_offsets;
  uint64_t blocks = (work + 255) / 256;
  if (blocks < 1) blocks = 1;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(reset_kernel, dim3((uint32_t)blocks), dim3(256), 0, stream, ctrl, states,
                     num_tiles, d_count, d_offsets, num_offsets);
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
  hipLaunchKernelGGL(build_tile_map_kernel, dim3(num_tensors), dim3(256), 0, stream, table,
                     tile_map);
  return hipGetLastError();
}

hipError_t launch_extract(const ExtractArgs& a, bool idx64, hipStream_t stream) {
  if (a.num_tiles == 0) return hipSuccess;
  const dim3 grid((uint32_t)a.num_tiles), block(kThreads);
  const bool multi = a.table != nullptr;
  if (idx64) {
    if (multi)
      hipLaunchKernelGGL((extract_kernel<int64_t, true>), grid, block, 0, stream, a);
    else
      hipLaunchKernelGGL((extract_kernel<int64_t, false>), grid, block, 0, stream, a);
  } else {
    if (multi)
      hipLaunchKernelGGL((extract_kernel<int32_t, true>), grid, block, 0, stream, a);
    else
      hipLaunchKernelGGL((extract_kernel<int32_t, false>), grid, block, 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace aurora
