// Write ceilings of the scatter that applies a delta, measured on the
// device the benchmark runs on (a measurement probe, not part of the
// library).  Prints one JSON line.
//
// Over a buffer of N words (the Qwen3-8B weight set's size) it times K
// stores at positions spaced like a 1% delta, pos(k) = k*B + (h(k) mod B)
// with B = N / K and h a fixed integer mix, i.e. about one entry per
// 64-byte line, with no loads of any index or value stream:
//   partial  one 2-byte non-temporal store per position, lane-strided the
//            way apply stores (a wavefront's store instruction covers 64
//            consecutive positions): each touched line costs one partial
//            write at the memory;
//   full     the whole aligned 64-byte line holding each position, written
//            by four lanes with 16-byte stores in one instruction: one full
//            line write per position.
// Rates are line writes per second (distinct touched lines / time); the
// median of 10 timed launches after 3 untimed ones.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <vector>

#define CHECK(x)                                                                 \
  do {                                                                           \
    hipError_t e_ = (x);                                                         \
    if (e_ != hipSuccess) {                                                      \
      std::fprintf(stderr, "%s:%d %s\n", __FILE__, __LINE__, hipGetErrorString(e_)); \
      std::exit(1);                                                              \
    }                                                                            \
  } while (0)

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) uint16_t g16;
typedef __attribute__((address_space(1))) u32x4 gv4;

__host__ __device__ inline uint32_t mix(uint64_t k) {
  uint64_t x = k * 0x9E3779B97F4A7C15ull;
  x ^= x >> 29;
  x *= 0xBF58476D1CE4E5B9ull;
  x ^= x >> 32;
  return (uint32_t)x;
}

// Position of entry k: below k*B + B <= K*B <= N, so every store is in bounds.
__host__ __device__ inline uint64_t pos_of(uint64_t k, uint64_t B) { return k * B + mix(k) % B; }

constexpr int kPerLane = 8;

__global__ __launch_bounds__(256) void partial_writes(uint16_t* w, uint64_t K, uint64_t B) {
  const uint32_t lane = threadIdx.x & 63;
  const uint64_t waves = (uint64_t)gridDim.x * 4;
  for (uint64_t wv = (uint64_t)blockIdx.x * 4 + (threadIdx.x >> 6); wv * 64 * kPerLane < K;
       wv += waves) {
#pragma unroll
    for (int u = 0; u < kPerLane; ++u) {
      const uint64_t k = wv * 64 * kPerLane + 64 * u + lane;
      if (k < K) __builtin_nontemporal_store((uint16_t)k, (g16*)(w + pos_of(k, B)));
    }
  }
}

// N is a multiple of 32 words, so the aligned line of any position is in bounds.
__global__ __launch_bounds__(256) void full_line_writes(uint16_t* w, uint64_t K, uint64_t B) {
  const uint64_t nth = (uint64_t)gridDim.x * 256;
  for (uint64_t t = (uint64_t)blockIdx.x * 256 + threadIdx.x; t < 4 * K; t += nth) {
    const uint64_t k = t >> 2;
    const uint64_t line = pos_of(k, B) >> 5;
    const u32x4 v = {(uint32_t)k, (uint32_t)k, (uint32_t)k, (uint32_t)k};
    __builtin_nontemporal_store(v, (gv4*)(w + line * 32 + 8 * (t & 3)));
  }
}

template <typename F>
static double median_ms(F&& launch) {
  hipEvent_t a, b;
  CHECK(hipEventCreate(&a));
  CHECK(hipEventCreate(&b));
  for (int i = 0; i < 3; ++i) launch();
  CHECK(hipDeviceSynchronize());
  std::vector<float> ms;
  for (int i = 0; i < 10; ++i) {
    CHECK(hipEventRecord(a, 0));
    launch();
    CHECK(hipEventRecord(b, 0));
    CHECK(hipEventSynchronize(b));
    float t = 0;
    CHECK(hipEventElapsedTime(&t, a, b));
    ms.push_back(t);
  }
  std::sort(ms.begin(), ms.end());
  CHECK(hipEventDestroy(a));
  CHECK(hipEventDestroy(b));
  return ms[ms.size() / 2];
}

int main() {
  const uint64_t N = 8190735360ull;   // words of the Qwen3-8B weight set (a multiple of 32)
  const uint64_t K = N / 100;
  const uint64_t B = N / K;
  // distinct 64-byte lines the positions touch (host count of the same formula)
  uint64_t lines = 0, last = ~0ull;
  for (uint64_t k = 0; k < K; ++k) {
    const uint64_t l = pos_of(k, B) >> 5;
    lines += l != last;
    last = l;
  }
  uint16_t* w = nullptr;
  CHECK(hipMalloc(&w, N * 2));
  CHECK(hipMemset(w, 0, N * 2));
  CHECK(hipDeviceSynchronize());
  const uint32_t gp = (uint32_t)std::min<uint64_t>(65536, (K + 2047) / 2048);
  const double tp = median_ms([&] { hipLaunchKernelGGL(partial_writes, dim3(gp), dim3(256), 0, 0, w, K, B); });
  const double tf = median_ms([&] { hipLaunchKernelGGL(full_line_writes, dim3(65536), dim3(256), 0, 0, w, K, B); });
  CHECK(hipGetLastError());
  CHECK(hipFree(w));
  std::printf("{\"words\": %llu, \"positions\": %llu, \"lines\": %llu, "
              "\"partial_ms\": %.4f, \"partial_line_writes_per_s\": %.1f, "
              "\"full_ms\": %.4f, \"full_line_writes_per_s\": %.1f}\n",
              (unsigned long long)N, (unsigned long long)K, (unsigned long long)lines, tp,
              lines / (tp * 1e-3), tf, lines / (tf * 1e-3));
  return 0;
}
