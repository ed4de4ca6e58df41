// Sparse delta extraction on gfx950: one pass over both bf16 copies that
// keeps every word whose bits changed and writes the kept positions and new
// words, in ascending position order, as two dense streams (AuroraRL
// Sec. 5.1, "Sparse encoding").
//
// Per workgroup (one tile of 8192 words):
//   1. take a tile id from a device counter (dynamic ids: a tile only ever
//      waits on tiles that were handed out earlier, hence already running);
//   2. read 16 bytes of each copy per lane per unrolled step;
//   3. compare 16-bit words, count changes per lane, turn the counts into
//      lane prefixes with four ballots + mbcnt (bit-sliced prefix sum);
//   4. combine wavefront totals through LDS into the tile's aggregate;
//   5. decoupled look-back over the tile-state array (Merrill & Garland,
//      "Single-pass Parallel Prefix Scan with Decoupled Look-back", 2016)
//      to learn how many kept words precede the tile;
//   6. write the kept (index, word) pairs at their final positions.
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

template <typename IdxT, bool kMulti>
__global__ __launch_bounds__(kThreads) void extract_kernel(ExtractArgs a) {
  __shared__ uint32_t s_tile;
  __shared__ uint32_t s_wave_total[kWaves];
  __shared__ uint64_t s_tile_excl;

  if (threadIdx.x == 0)
    s_tile = __hip_atomic_fetch_add(&a.ctrl->tile_counter, 1u, __ATOMIC_RELAXED,
                                    __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  const uint64_t tile = s_tile;
  const TensorDesc d = kMulti ? a.table[a.tile_map[tile]] : a.single;
  const uint64_t local_tile = tile - d.first_tile;

  const uint32_t lane = lane_id();
  const uint32_t wave = threadIdx.x >> 6;
  const int64_t g0 = (int64_t)(local_tile * kGroupsPerTile) + wave * kGroupsPerWave + lane;

  u32x4 p[kChunks], q[kChunks];
#pragma unroll
  for (int u = 0; u < kChunks; ++u) load_group(d, g0 + 64 * u, p[u], q[u]);

  uint32_t mask[kChunks];
  uint32_t lane_prefix[kChunks];
  uint32_t chunk_base[kChunks];   // wave-uniform: kept words of earlier chunks
  uint32_t wave_total = 0;
#pragma unroll
  for (int u = 0; u < kChunks; ++u) {
    mask[u] = changed_mask(p[u], q[u]);
    const uint32_t c = __popc(mask[u]);
    const uint64_t b0 = __ballot(c & 1), b1 = __ballot(c & 2);
    const uint64_t b2 = __ballot(c & 4), b3 = __ballot(c & 8);
    lane_prefix[u] = mbcnt64(b0) + 2 * mbcnt64(b1) + 4 * mbcnt64(b2) + 8 * mbcnt64(b3);
    chunk_base[u] = wave_total;
    wave_total += __popcll(b0) + 2 * __popcll(b1) + 4 * __popcll(b2) + 8 * __popcll(b3);
  }
  if (lane == 0) s_wave_total[wave] = wave_total;
  __syncthreads();

  uint32_t wave_excl = 0, tile_total = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const uint32_t t = s_wave_total[w];
    wave_excl += (w < (int)wave) ? t : 0u;
    tile_total += t;
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
        uint64_t st, need, prefix_lanes;
        for (;;) {
          st = (t >= 0) ? load_state(&a.states[t]) : kStatePrefix;
          const uint64_t empty = __ballot((st & kStateFlagMask) == kStateEmpty);
          prefix_lanes = __ballot((st & kStateFlagMask) == kStatePrefix);
          // lanes that count: up to and including the nearest full prefix
          need = prefix_lanes ? (((prefix_lanes & (0 - prefix_lanes)) << 1) - 1) : ~0ull;
          if ((empty & need) == 0) break;
          __builtin_amdgcn_s_sleep(1);
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

  // Scatter-free write: every kept word goes to its final slot.
  IdxT* out_idx = reinterpret_cast<IdxT*>(a.out_idx);
#pragma unroll
  for (int u = 0; u < kChunks; ++u) {
    uint32_t m = mask[u];
    if (m == 0) continue;
    uint64_t pos = tile_excl + wave_excl + chunk_base[u] + lane_prefix[u];
    const int64_t e0 = 8 * (g0 + 64 * u) - (int64_t)d.head;
    while (m) {
      const int j = __builtin_ctz(m);
      m &= m - 1;
      if (pos < a.capacity) {
        const uint32_t dw = q[u][j >> 1];
        out_idx[pos] = (IdxT)((int64_t)d.base + e0 + j);
        a.out_val[pos] = (uint16_t)((j & 1) ? (dw >> 16) : (dw & 0xFFFFu));
      }
      ++pos;
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
    ctrl->tile_counter = 0;
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
