// Delta application on gfx950: write each kept word back into the flat
// storage of the rollout copy, w[idx[k]] = val[k] (AuroraRL Sec. 5.1 and
// Sec. 5.2: an in-place flat scatter at an end-of-batch safe point).
//
// The value stream holds the new words themselves, so the scatter assigns
// rather than adds: the result is bit-exact and applying a delta twice
// changes nothing.  Indices are distinct, so no two lanes write one word
// and no atomics are needed.  The index and value streams are read with
// 16-byte loads (8 entries per lane); the 2-byte stores are scattered.
#include "delta_internal.h"

namespace aurora {

constexpr int kApplyThreads = 256;
constexpr int kApplyPerLane = 8;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void flag_error(uint32_t* err) {
  if (err) __hip_atomic_fetch_or(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <typename IdxT>
__device__ __forceinline__ void load8(const IdxT* idx, const uint16_t* val, uint64_t k0,
                                      uint64_t count, bool vec, int64_t (&i)[8],
                                      uint16_t (&v)[8], int& valid) {
  if (vec && k0 + 8 <= count) {
    const u32x4 vv = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(val + k0));
#pragma unroll
    for (int j = 0; j < 8; ++j)
      v[j] = (uint16_t)((j & 1) ? (vv[j >> 1] >> 16) : (vv[j >> 1] & 0xFFFFu));
    if (sizeof(IdxT) == 8) {
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const u32x4 x = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(idx + k0) + h);
        i[2 * h] = (int64_t)(((uint64_t)x[1] << 32) | x[0]);
        i[2 * h + 1] = (int64_t)(((uint64_t)x[3] << 32) | x[2]);
      }
    } else {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const u32x4 x = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(idx + k0) + h);
#pragma unroll
        for (int j = 0; j < 4; ++j) i[4 * h + j] = (int64_t)(int32_t)x[j];
      }
    }
    valid = 8;
  } else {
    valid = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (k0 + j < count) {
        i[j] = (int64_t)idx[k0 + j];
        v[j] = val[k0 + j];
        valid = j + 1;
      }
    }
  }
}

template <typename IdxT>
__global__ __launch_bounds__(kApplyThreads) void apply_kernel(uint16_t* __restrict__ w, uint64_t n,
                                                              const IdxT* __restrict__ idx,
                                                              const uint16_t* __restrict__ val,
                                                              uint64_t count, uint32_t* err,
                                                              bool vec) {
  const uint64_t stride = (uint64_t)gridDim.x * kApplyThreads * kApplyPerLane;
  for (uint64_t k0 = ((uint64_t)blockIdx.x * kApplyThreads + threadIdx.x) * kApplyPerLane;
       k0 < count; k0 += stride) {
    int64_t i[8];
    uint16_t v[8];
    int valid;
    load8(idx, val, k0, count, vec, i, v, valid);
    bool bad = false;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (j < valid) {
        if (i[j] >= 0 && (uint64_t)i[j] < n)
          w[i[j]] = v[j];
        else
          bad = true;
      }
    }
    if (bad) flag_error(err);
  }
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
    uint32_t* err, bool vec) {
  const uint64_t stride = (uint64_t)gridDim.x * kApplyThreads * kApplyPerLane;
  const uint64_t total = bases[T];
  for (uint64_t k0 = ((uint64_t)blockIdx.x * kApplyThreads + threadIdx.x) * kApplyPerLane;
       k0 < count; k0 += stride) {
    int64_t i[8];
    uint16_t v[8];
    int valid;
    load8(idx, val, k0, count, vec, i, v, valid);
    bool bad = false;
    uint32_t t = 0;
    uint64_t lo = 1, hi = 0;   // empty range: forces a search first
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (j < valid) {
        const int64_t g = i[j];
        if (g < 0 || (uint64_t)g >= total) {
          bad = true;
          continue;
        }
        if (!((uint64_t)g >= lo && (uint64_t)g < hi)) {
          t = find_tensor(bases, T, (uint64_t)g);
          lo = bases[t];
          hi = bases[t + 1];
        }
        ptrs[t][(uint64_t)g - lo] = v[j];
      }
    }
    if (bad) flag_error(err);
  }
}

static uint32_t apply_blocks(uint64_t count) {
  const uint64_t per_block = (uint64_t)kApplyThreads * kApplyPerLane;
  uint64_t blocks = (count + per_block - 1) / per_block;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  return (uint32_t)blocks;
}

hipError_t launch_apply(uint16_t* w, uint64_t n, bool idx64, const void* idx,
                        const uint16_t* val, uint64_t count, uint32_t* err,
                        hipStream_t stream) {
  if (count == 0) return hipSuccess;
  const bool vec = ((uintptr_t)idx % 16 == 0) && ((uintptr_t)val % 16 == 0);
  if (idx64)
    hipLaunchKernelGGL(apply_kernel<int64_t>, dim3(apply_blocks(count)), dim3(kApplyThreads), 0,
                       stream, w, n, (const int64_t*)idx, val, count, err, vec);
  else
    hipLaunchKernelGGL(apply_kernel<int32_t>, dim3(apply_blocks(count)), dim3(kApplyThreads), 0,
                       stream, w, n, (const int32_t*)idx, val, count, err, vec);
  return hipGetLastError();
}

hipError_t launch_apply_multi(const uint64_t* bases, uint16_t* const* ptrs, uint32_t T,
                              const int64_t* idx, const uint16_t* val, uint64_t count,
                              uint32_t* err, hipStream_t stream) {
  if (count == 0) return hipSuccess;
  const bool vec = ((uintptr_t)idx % 16 == 0) && ((uintptr_t)val % 16 == 0);
  hipLaunchKernelGGL(apply_multi_kernel, dim3(apply_blocks(count)), dim3(kApplyThreads), 0, stream,
                     bases, ptrs, T, idx, val, count, err, vec);
  return hipGetLastError();
}

}  // namespace aurora
