// Delta application on gfx950: write each kept word back into the flat
// storage of the rollout copy, w[idx[k]] = val[k] (AuroraRL Sec. 5.1 and
// Sec. 5.2: an in-place flat scatter at an end-of-batch safe point).
//
// The value stream holds the new words themselves, so the scatter assigns
// rather than adds: the result is bit-exact and applying a delta twice
// changes nothing.  Indices are distinct, so no two lanes write one word
// and no atomics are needed.
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

__device__ __forceinline__ void store_word(uint16_t* p, uint16_t v) {
  if (kNtScatter)
    __builtin_nontemporal_store(v, p);
  else
    *p = v;
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

}  // namespace aurora
