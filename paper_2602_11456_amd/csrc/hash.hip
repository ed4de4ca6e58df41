// Integrity hashing of delta checkpoints on gfx950 (AuroraRL Sec. 5.1: every
// delta checkpoint is an immutable versioned file with an integrity hash;
// Sec. 5.2: it travels as segments that are verified against that hash).
//
// The hash is XXH64 (Y. Collet, xxHash specification), computed by four
// lanes per segment: lane q keeps accumulator q and reads the q-th 8-byte
// word of every 32-byte stripe, so a wavefront hashes 16 segments at once
// and each load instruction reads 32 contiguous bytes per segment.  Lane 0
// of the quad then merges the four accumulators, folds in the tail (fewer
// than 32 bytes) and applies the final avalanche.
//
// The artifact (header, tensor table, index stream, value stream, segment
// hash table) is laid out by artifact_layout; its hash is the XXH64 of the
// segment hash table seeded with the XXH64 of the header's first 80 bytes,
// so it covers the header fields, and through the table every payload byte.
#include "delta_internal.h"
#include "hash.h"

namespace aurora {

constexpr uint64_t kP1 = 11400714785074694791ull;
constexpr uint64_t kP2 = 14029467366897019727ull;
constexpr uint64_t kP3 = 1609587929392839161ull;
constexpr uint64_t kP4 = 9650029242287828579ull;
constexpr uint64_t kP5 = 2870177450012600261ull;

__device__ __forceinline__ uint64_t rotl(uint64_t x, int r) { return (x << r) | (x >> (64 - r)); }
__device__ __forceinline__ uint64_t xx_round(uint64_t acc, uint64_t lane) {
  return rotl(acc + lane * kP2, 31) * kP1;
}
__device__ __forceinline__ uint64_t ld_le64(const uint8_t* p) {
  uint64_t v = 0;
#pragma unroll
  for (int b = 7; b >= 0; --b) v = (v << 8) | p[b];
  return v;
}

// XXH64 of [p, p + len) by the quad of lanes that this lane belongs to (q =
// its position in the quad; all four lanes call it with the same p, len,
// seed).  p + 8 must be 8-aligned... p itself 8-aligned.  The result is
// valid in every lane of the quad.
__device__ __forceinline__ uint64_t xxh64_quad(const uint8_t* p, uint64_t len, uint64_t seed,
                                               uint32_t q, bool active) {
  const uint64_t stripes = active ? len / 32 : 0;
  uint64_t acc = q == 0 ? seed + kP1 + kP2 : q == 1 ? seed + kP2 : q == 2 ? seed : seed - kP1;
  const uint64_t* w = (const uint64_t*)p + q;
  uint64_t s = 0;
  for (; s + 4 <= stripes; s += 4) {
    const uint64_t x0 = w[4 * s], x1 = w[4 * s + 4], x2 = w[4 * s + 8], x3 = w[4 * s + 12];
    acc = xx_round(acc, x0);
    acc = xx_round(acc, x1);
    acc = xx_round(acc, x2);
    acc = xx_round(acc, x3);
  }
  for (; s < stripes; ++s) acc = xx_round(acc, w[4 * s]);
  const uint32_t base = (threadIdx.x & 63) & ~3u;
  const uint64_t a1 = __shfl(acc, base), a2 = __shfl(acc, base + 1), a3 = __shfl(acc, base + 2),
                 a4 = __shfl(acc, base + 3);
  uint64_t h;
  if (len >= 32) {
    h = rotl(a1, 1) + rotl(a2, 7) + rotl(a3, 12) + rotl(a4, 18);
    h = (h ^ xx_round(0, a1)) * kP1 + kP4;
    h = (h ^ xx_round(0, a2)) * kP1 + kP4;
    h = (h ^ xx_round(0, a3)) * kP1 + kP4;
    h = (h ^ xx_round(0, a4)) * kP1 + kP4;
  } else {
    h = seed + kP5;
  }
  h += len;
  if (active) {   // the tail, the same in every lane
    const uint8_t* t = p + 32 * (len / 32);
    uint64_t left = len % 32;
    while (left >= 8) {
      h ^= xx_round(0, ld_le64(t));
      h = rotl(h, 27) * kP1 + kP4;
      t += 8;
      left -= 8;
    }
    if (left >= 4) {
      const uint64_t v = (uint64_t)t[0] | ((uint64_t)t[1] << 8) | ((uint64_t)t[2] << 16) |
                         ((uint64_t)t[3] << 24);
      h ^= v * kP1;
      h = rotl(h, 23) * kP2 + kP3;
      t += 4;
      left -= 4;
    }
    while (left >= 1) {
      h ^= (uint64_t)(*t) * kP5;
      h = rotl(h, 11) * kP1;
      ++t;
      --left;
    }
  }
  h ^= h >> 33;
  h *= kP2;
  h ^= h >> 29;
  h *= kP3;
  h ^= h >> 32;
  return h;
}

// out[s] = XXH64 of segment s (seg_bytes each, the last one shorter).
__global__ __launch_bounds__(256) void xxh64_segments_kernel(const uint8_t* data, uint64_t nbytes,
                                                             uint64_t seg_bytes, uint64_t seed,
                                                             uint64_t nsegs, uint64_t* out) {
  const uint64_t g = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const uint64_t seg = g >> 2;
  const uint32_t q = g & 3;
  const bool active = seg < nsegs;
  const uint64_t off = active ? seg * seg_bytes : 0;
  const uint64_t len = active ? (nbytes - off < seg_bytes ? nbytes - off : seg_bytes) : 0;
  const uint64_t h = xxh64_quad(data + off, len, seed, q, active);
  if (active && q == 0) out[seg] = h;
}

// Artifact hash: XXH64(table, seed = XXH64(header[0, 80), 0)); written into
// the header (seal) or compared with it (verify).  One quad.
__global__ void artifact_hash_kernel(uint8_t* art, uint64_t hashes_off, uint64_t nsegs,
                                     bool seal, uint32_t* d_header_bad) {
  const uint32_t q = threadIdx.x & 3;
  const uint64_t h0 = xxh64_quad(art, kArtifactHashedHeader, 0, q, true);
  const uint64_t h = xxh64_quad(art + hashes_off, 8 * nsegs, h0, q, true);
  if (threadIdx.x == 0) {
    uint64_t* field = (uint64_t*)(art + kArtifactHashField);
    if (seal)
      *field = h;
    else
      *d_header_bad = *field != h;
  }
}

// The header (by value) into the artifact.
__global__ void artifact_header_kernel(uint8_t* art, delta_artifact_header_t h) {
  const uint8_t* src = (const uint8_t*)&h;
  for (uint32_t i = threadIdx.x; i < sizeof(h); i += blockDim.x) art[i] = src[i];
}

// Counts the segments whose stored hash differs from the recomputed one.
__global__ void artifact_compare_kernel(const uint64_t* stored, const uint64_t* fresh,
                                        uint64_t nsegs, unsigned long long* d_bad,
                                        unsigned long long* d_first_bad) {
  const uint64_t s = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (s < nsegs && stored[s] != fresh[s]) {
    atomicAdd(d_bad, 1ull);
    if (d_first_bad) atomicMin(d_first_bad, (unsigned long long)s);
  }
}

__global__ void artifact_verify_init_kernel(unsigned long long* d_bad,
                                            unsigned long long* d_first_bad) {
  *d_bad = 0;
  if (d_first_bad) *d_first_bad = ~0ull;
}

hipError_t launch_hash_segments(const uint8_t* data, uint64_t nbytes, uint64_t seg_bytes,
                                uint64_t seed, uint64_t* out, hipStream_t stream) {
  const uint64_t nsegs = nbytes ? (nbytes + seg_bytes - 1) / seg_bytes : 0;
  if (nsegs == 0) return hipSuccess;
  const uint64_t threads = 4 * nsegs;
  hipLaunchKernelGGL(xxh64_segments_kernel, dim3((uint32_t)((threads + 255) / 256)), dim3(256), 0,
                     stream, data, nbytes, seg_bytes, seed, nsegs, out);
  return hipGetLastError();
}

ArtifactLayout artifact_layout(uint64_t num_tensors, uint64_t count, uint64_t idx_bytes,
                               uint64_t seg_bytes) {
  ArtifactLayout L;
  L.table = sizeof(delta_artifact_header_t);
  L.idx = L.table + 24 * num_tensors;
  L.val = align_up(L.idx + idx_bytes, 8);
  L.hashes = align_up(L.val + 2 * count, 8);
  const uint64_t hashed = L.hashes - L.table;
  L.num_segments = seg_bytes ? (hashed + seg_bytes - 1) / seg_bytes : 0;
  L.total = L.hashes + 8 * L.num_segments;
  return L;
}

// The artifact's tensor table (one row {words, first entry, first index
// byte} per tensor) and the zero padding that aligns the value stream and
// the hash table: every byte of [table, hashes) is then written, so the
// segment hashes do not depend on what the buffer held before.
__global__ __launch_bounds__(256) void artifact_table_kernel(uint8_t* art, ArtifactLayout L,
                                                             const uint64_t* numels,
                                                             const uint64_t* offs,
                                                             const uint64_t* byte_offs,
                                                             uint32_t T, uint64_t idx_bytes,
                                                             uint64_t count) {
  uint64_t* rows = (uint64_t*)(art + L.table);
  for (uint32_t t = blockIdx.x * blockDim.x + threadIdx.x; t < T; t += gridDim.x * blockDim.x) {
    rows[3 * (uint64_t)t + 0] = numels[t];
    rows[3 * (uint64_t)t + 1] = offs[t];
    rows[3 * (uint64_t)t + 2] = byte_offs ? byte_offs[t] : 8 * offs[t];
  }
  if (blockIdx.x == 0 && threadIdx.x < 8) {
    const uint64_t a = L.idx + idx_bytes, b = L.val + 2 * count;
    if (a + threadIdx.x < L.val) art[a + threadIdx.x] = 0;
    if (b + threadIdx.x < L.hashes) art[b + threadIdx.x] = 0;
  }
}

hipError_t launch_artifact_table(uint8_t* art, const ArtifactLayout& L, const uint64_t* numels,
                                 const uint64_t* offs, const uint64_t* byte_offs, uint32_t T,
                                 uint64_t idx_bytes, uint64_t count, hipStream_t stream) {
  const uint32_t blocks = T ? (T + 255) / 256 : 1;
  hipLaunchKernelGGL(artifact_table_kernel, dim3(blocks < 64 ? blocks : 64), dim3(256), 0, stream,
                     art, L, numels, offs, byte_offs, T, idx_bytes, count);
  return hipGetLastError();
}

hipError_t launch_artifact_seal(uint8_t* art, const ArtifactLayout& L,
                                const delta_artifact_header_t& h, hipStream_t stream) {
  hipLaunchKernelGGL(artifact_header_kernel, dim3(1), dim3(128), 0, stream, art, h);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = launch_hash_segments(art + L.table, L.hashes - L.table, h.seg_bytes, h.version,
                           (uint64_t*)(art + L.hashes), stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(artifact_hash_kernel, dim3(1), dim3(64), 0, stream, art, L.hashes,
                     L.num_segments, true, (uint32_t*)nullptr);
  return hipGetLastError();
}

hipError_t launch_artifact_verify(const uint8_t* art, const ArtifactLayout& L, uint64_t seg_bytes,
                                  uint64_t seed, uint64_t* fresh, uint64_t* d_bad,
                                  uint64_t* d_first_bad, uint32_t* d_header_bad,
                                  hipStream_t stream) {
  hipLaunchKernelGGL(artifact_verify_init_kernel, dim3(1), dim3(1), 0, stream,
                     (unsigned long long*)d_bad, (unsigned long long*)d_first_bad);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = launch_hash_segments(art + L.table, L.hashes - L.table, seg_bytes, seed, fresh, stream);
  if (e != hipSuccess) return e;
  if (L.num_segments) {
    hipLaunchKernelGGL(artifact_compare_kernel, dim3((uint32_t)((L.num_segments + 255) / 256)),
                       dim3(256), 0, stream, (const uint64_t*)(art + L.hashes), fresh,
                       L.num_segments, (unsigned long long*)d_bad,
                       (unsigned long long*)d_first_bad);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(artifact_hash_kernel, dim3(1), dim3(64), 0, stream, (uint8_t*)art, L.hashes,
                     L.num_segments, false, d_header_bad);
  return hipGetLastError();
}

}  // namespace aurora
