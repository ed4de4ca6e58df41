// Chunked extraction with the output streamed to pinned host memory
// (AuroraRL Sec. 5.2, "Overlapped extraction and transfer": the delta is cut
// into segments that are emitted as soon as each is encoded, striped
// round-robin over several parallel channels).
//
// The global index space of the tensor list is cut into chunks of
// `chunk_elems` words; a chunk may span several tensors and start inside
// one.  Chunk c is extracted into staging slot c mod S (S streams, S slots).
// Three streams have roles: streams[0] reads, running every chunk's stage
// kernel (the pass over both copies) back to back; streams[1] codes,
// taking the kernels that finish each chunk (its finalize pass, and for
// the coded form the group records before it) once its stage kernel is
// done, while the next chunk is being read; streams[2] delivers the chunks
// in order: one kernel per chunk (plain, with four or more slots, per two
// chunks) reads the counts and the running totals from device memory and
// stores the entries straight into the pinned host arrays over the host
// link (kernel stores into pinned memory reach the 55 GB/s of DMA copies
// and need no host round trip per chunk).  Coded, the extract writes the
// chunk's positions gap + LEB128 coded instead of as indices (no index
// stream in between).  A delivery waits on its chunk's coding; the reading of a chunk
// that reuses a slot waits on the delivery of the slot's previous chunk.
// The host only enqueues and waits once, at the end.  With S == 2 reading
// and coding share streams[0]; with S == 1 everything runs in order on it.

#include <string.h>

#include <vector>

#include "aurora_delta.h"
#include "delta_internal.h"

using namespace aurora;

namespace {

// Slices of chunk [lo, hi) of the global index space.
void chunk_slices(const uint16_t* const* prevs, const uint16_t* const* nexts,
                  const uint64_t* numels, int32_t T, uint64_t lo, uint64_t hi,
                  std::vector<SliceIn>& out) {
  out.clear();
  uint64_t base = 0;
  for (int32_t t = 0; t < T && base < hi; ++t) {
    const uint64_t n = numels[t];
    const uint64_t a = lo > base ? lo : base;
    const uint64_t b = hi < base + n ? hi : base + n;
    if (a < b)
      out.push_back({prevs[t] + (a - base), nexts[t] + (a - base), b - a, a, (uint32_t)t, base});
    base += n;
  }
}


struct StagingLayout {
  size_t idx, val, count, nbytes, bytes, ws, ws_bytes, per_stream;
  size_t run, chunk_counts, total;   // after the S slots: running totals, per-chunk counts
};

// Longest LEB128 code of a number below `chunk` (every gap inside a chunk,
// and its first index relative to the chunk start, is below the chunk size).
uint64_t leb_bytes_per_entry(uint64_t chunk) {
  uint64_t v = chunk > 0 ? chunk - 1 : 0, n = 1;
  while (v >= 128) {
    v >>= 7;
    ++n;
  }
  return n;
}

// Coded, a slot holds no index stream: the extract writes the code itself.
StagingLayout staging_layout(uint64_t chunk, size_t ws_bytes, bool leb, int streams,
                             uint64_t nchunks) {
  StagingLayout L;
  L.idx = 0;
  L.val = align_up(L.idx + (leb ? 0 : 8 * chunk));
  L.count = align_up(L.val + 2 * chunk);
  L.nbytes = L.count + 8;
  L.bytes = align_up(L.nbytes + 8);
  L.ws = align_up(L.bytes + (leb ? leb_bytes_per_entry(chunk) * chunk : 0));
  L.ws_bytes = ws_bytes;
  L.per_stream = align_up(L.ws + ws_bytes);
  L.run = L.per_stream * (size_t)streams;
  L.chunk_counts = align_up(L.run + 4 * sizeof(uint64_t));
  L.total = align_up(L.chunk_counts + sizeof(uint64_t) * nchunks);
  return L;
}

// Device address of a pinned host range, or nullptr if [h, h + bytes) is
// not pinned host memory the device can reach.
void* host_range_on_device(const void* h, size_t bytes) {
  if (!h || bytes == 0) return nullptr;
  void* d0 = nullptr;
  void* d1 = nullptr;
  if (hipHostGetDevicePointer(&d0, const_cast<void*>(h), 0) != hipSuccess ||
      hipHostGetDevicePointer(&d1, (char*)const_cast<void*>(h) + bytes - 1, 0) != hipSuccess ||
      (char*)d1 - (char*)d0 != (ptrdiff_t)(bytes - 1)) {
    (void)hipGetLastError();   // do not leave the lookup's error behind
    return nullptr;
  }
  return d0;
}

// One delivery: the entries (and coded bytes) of one chunk, or of two
// consecutive chunks, from their staging slots to the host arrays at the
// running totals, which sit in device memory, double-buffered by the
// delivery's ordinal k (every thread reads run[k & 1]; thread 0 writes
// run[(k + 1) & 1]).  Entries past a host array's capacity are dropped;
// the totals stay true.
struct DeliverChunk {
  const int64_t* idx;
  const uint16_t* val;
  const uint8_t* bytes;        // coded, else nullptr
  const uint64_t* d_count;     // entries of the chunk
  const uint64_t* d_nbytes;    // coded: code bytes of the chunk
};
struct DeliverArgs {
  DeliverChunk ch[2];
  uint32_t n;                  // chunks delivered: 1 or 2
  uint64_t c;                  // the first of them
  uint64_t k;                  // ordinal of this delivery
  uint64_t* run;               // [2][2] (entries, bytes)
  uint64_t* chunk_counts;      // coded: entry count of every chunk
  int64_t* h_idx;              // device views of the pinned host arrays
  uint64_t h_idx_cap;
  uint8_t* h_bytes;
  uint64_t h_bytes_cap;
  uint16_t* h_val;
  uint64_t h_val_cap;
  uint32_t xcds;               // workgroups on the last `xcds` XCDs store
};

// Streams beyond the three roles stay idle: a process gets four hardware
// queues by default, and streams beyond that share a queue, which
// serialises their work.
// Stores into host memory are slow to complete, and while many are
// outstanding the GPU's HBM reads slow down: a host-write kernel spread over
// all 8 XCDs cut a concurrent HBM read kernel from 6.9 to 1.8 TB/s.  So the
// delivery runs few workgroups, on the last XCDs (workgroup b runs on XCD
// b mod 8; the grid holds the same count per XCD and only those on the
// last `xcds` work; small kernels of one or a few workgroups, such as the
// scans, run on the first XCDs).  How few is a trade between filling the
// host link and leaving the reads alone (Qwen3-14B, 2^27-word chunks,
// plain / coded ms): 2 XCDs x 8 workgroups 30.4 / 17.1; 4 x 4 29.7 / 17.2;
// 8 x 2 29.7-29.8 / 17.0; 1 x 4 35.0 / 13.7-14.5; 2 x 2 34.4 / 14.0;
// 1 x 2 37.4 / 18.6; plain 4 x 5 / 4 x 6 / 4 x 8 / 3 x 6 / 6 x 4 29.4 /
// 29.2-29.4 / 32.4 / 29.8 / 34.5; coded 1 x 3 / 1 x 5 / 1 x 6 / 1 x 7 /
// 1 x 8 / 2 x 4 16.3 / 13.7 / 13.3-13.5 / 13.9 / 14.4 / 15.2.  Once the
// finalize pass scanned for itself, a second sweep (same order of runs)
// gave plain 4 x 6 / 2 x 6 / 2 x 8 / 1 x 8 / 1 x 12 / 1 x 16 30.4 / 29.8 /
// 29.8 / 31.1 / 30.4 / 30.5 and coded 1 x 6 / 2 x 3 / 1 x 4 / 1 x 8 /
// 1 x 10 / 1 x 12 13.3-13.5 / 13.7-13.8 / 14.6 / 14.2 / 15.4 / 15.7.  The
// plain stream (10 bytes per entry) needs the link's rate and takes 2 x 6;
// the coded one (about 3.3) far less.  Its chunks are small (about 4.4 MB),
// and a workgroup's rounds of loads wait on the reads beside them, so the
// bytes each round keeps in flight matter as much as the workgroup count:
// coded 1 x 3 workgroups of 512 threads with 8 vectors per thread per
// round 12.4-12.7 ms, against 13.3-13.5 for 1 x 6 of 256 threads with 4
// (1 x 2 / 1 x 4 of 512 x 8: 15.8 / 13.8; 1 x 3 of 512 x 16: 12.9; 1 x 3
// of 256 x 8 / 1024 x 8: 15.5 / 14.5; 1 x 6 of 256 x 8 / 256 x 16 / 512 x
// 4: 14.2 / 15.2 / 15.3).  The plain kind measured 29.8-30.5 ms in every
// one of these forms and keeps 256 threads with 4.
constexpr int kXcds = 8;
struct DeliverShape {
  uint32_t xcds, per_xcd;
};
constexpr DeliverShape kDeliverPlain = {2, 6};
constexpr DeliverShape kDeliverCoded = {1, 3};
constexpr int kPlainThreads = 256, kPlainUnroll = 4;
constexpr int kCodedThreads = 512, kCodedUnroll = 8;

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
// four dwords at a 4-byte aligned address (one 16-byte load)
typedef uint32_t u32x4a_t __attribute__((ext_vector_type(4), aligned(4)));

// dst[0, n) = src[0, n) by the whole grid, where src is 4-byte aligned and
// readable up to 4 bytes past n, and dst (host memory) has any alignment:
// the bytes before dst's first 16-byte boundary and after its last one are
// stored one by one; in between every store is a whole aligned 16 bytes,
// assembled from five aligned source dwords with byte-aligning shifts.
template <int kCopyUnroll>
__device__ void copy_bytes(uint8_t* dst, const uint8_t* src, uint64_t n, uint64_t i0,
                           uint64_t stride) {
  uint64_t head = (16 - ((uintptr_t)dst & 15)) & 15;
  if (head > n) head = n;
  const uint64_t body = (n - head) / 16;
  const uint64_t tail0 = head + 16 * body;
  for (uint64_t k = i0; k < head; k += stride) dst[k] = src[k];
  for (uint64_t k = tail0 + i0; k < n; k += stride) dst[k] = src[k];
  const uint32_t shift = (uint32_t)(head & 3);
  const uint32_t* s32 = reinterpret_cast<const uint32_t*>(src + (head & ~(uint64_t)3));
  u32x4_t* d16 = reinterpret_cast<u32x4_t*>(dst + head);
  // kCopyUnroll vectors per thread per round, all loaded before any store,
  // so that the loads' latency overlaps
  for (uint64_t j0 = i0; j0 < body; j0 += kCopyUnroll * stride) {
    u32x4a_t w[kCopyUnroll];
    uint32_t w4[kCopyUnroll];
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) {
      const uint64_t j = j0 + u * stride;
      w[u] = j < body ? *reinterpret_cast<const u32x4a_t*>(s32 + 4 * j) : u32x4a_t{0, 0, 0, 0};
      w4[u] = (j < body && shift) ? s32[4 * j + 4] : 0u;
    }
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) {
      const uint64_t j = j0 + u * stride;
      if (j >= body) break;
      u32x4_t v;
      if (shift) {
        // byte `shift` onwards of each 8-byte pair (hi:lo)
        v[0] = __builtin_amdgcn_alignbyte(w[u][1], w[u][0], shift);
        v[1] = __builtin_amdgcn_alignbyte(w[u][2], w[u][1], shift);
        v[2] = __builtin_amdgcn_alignbyte(w[u][3], w[u][2], shift);
        v[3] = __builtin_amdgcn_alignbyte(w4[u], w[u][3], shift);
      } else {
        v = u32x4_t{w[u][0], w[u][1], w[u][2], w[u][3]};
      }
      __builtin_nontemporal_store(v, d16 + j);
    }
  }
}

// kThreads threads per workgroup, each with kUnroll 16-byte vectors in
// flight per round.
template <int kThreads, int kUnroll>
__global__ __launch_bounds__(kThreads) void deliver_kernel(DeliverArgs a) {
  uint64_t cnt[2] = {0, 0}, nb[2] = {0, 0};
  for (uint32_t j = 0; j < a.n; ++j) {
    cnt[j] = *a.ch[j].d_count;
    nb[j] = a.ch[j].bytes ? *a.ch[j].d_nbytes : 0;
  }
  const uint64_t* r = a.run + 2 * (a.k & 1);
  const uint64_t be0 = r[0], bb0 = r[1];
  const uint32_t xcd = blockIdx.x % kXcds;
  const uint32_t first_xcd = kXcds - a.xcds;
  if (xcd < first_xcd) return;
  const uint64_t wg = (uint64_t)(blockIdx.x / kXcds) * a.xcds + (xcd - first_xcd);
  const uint64_t i0 = wg * blockDim.x + threadIdx.x;
  const uint64_t stride = (uint64_t)(gridDim.x / kXcds) * a.xcds * blockDim.x;
  if (i0 == 0) {
    uint64_t* w = a.run + 2 * ((a.k + 1) & 1);
    w[0] = be0 + cnt[0] + cnt[1];
    w[1] = bb0 + nb[0] + nb[1];
    if (a.chunk_counts)
      for (uint32_t j = 0; j < a.n; ++j) a.chunk_counts[a.c + j] = cnt[j];
  }
  uint64_t be = be0, bb = bb0;
  for (uint32_t j = 0; j < a.n; ++j) {
    const DeliverChunk& ch = a.ch[j];
    const uint64_t ne = be < a.h_val_cap ? (a.h_val_cap - be < cnt[j] ? a.h_val_cap - be : cnt[j]) : 0;
    copy_bytes<kUnroll>((uint8_t*)(a.h_val + be), (const uint8_t*)ch.val, 2 * ne, i0, stride);
    if (a.h_idx) {
      const uint64_t ni =
          be < a.h_idx_cap ? (a.h_idx_cap - be < cnt[j] ? a.h_idx_cap - be : cnt[j]) : 0;
      copy_bytes<kUnroll>((uint8_t*)(a.h_idx + be), (const uint8_t*)ch.idx, 8 * ni, i0, stride);
    }
    if (ch.bytes) {
      const uint64_t n =
          bb < a.h_bytes_cap ? (a.h_bytes_cap - bb < nb[j] ? a.h_bytes_cap - bb : nb[j]) : 0;
      copy_bytes<kUnroll>(a.h_bytes + bb, ch.bytes, n, i0, stride);
    }
    be += cnt[j];
    bb += nb[j];
  }
}

__global__ void run_reset_kernel(uint64_t* run) {
  if (threadIdx.x < 4) run[threadIdx.x] = 0;
}

// Largest workspace any chunk's extract needs (tiles at worst alignment).
size_t max_chunk_workspace(const uint64_t* numels, int32_t T, uint64_t total, uint64_t chunk,
                           bool coded) {
  size_t best = 0;
  for (uint64_t lo = 0; lo < total; lo += chunk) {
    const uint64_t hi = (total - lo < chunk) ? total : lo + chunk;
    uint64_t tiles = 0, rows = 0, base = 0;
    for (int32_t t = 0; t < T && base < hi; ++t) {
      const uint64_t a = lo > base ? lo : base;
      const uint64_t b = hi < base + numels[t] ? hi : base + numels[t];
      if (a < b) {
        tiles += tiles_bound(b - a);
        ++rows;
      }
      base += numels[t];
    }
    const size_t need = workspace_bytes(tiles, rows, kDefaultStageCap, coded);
    if (need > best) best = need;
  }
  return best;
}

}  // namespace

extern "C" {

static size_t staging_bytes_impl(const uint64_t* numels, int32_t num_tensors,
                                 const delta_pipeline_opts_t* opts, bool leb) {
  if (!opts || opts->chunk_elems == 0 || opts->num_streams < 1 || opts->num_streams > 16 ||
      num_tensors < 0 || (num_tensors > 0 && !numels))
    return 0;
  uint64_t total = 0;
  for (int32_t t = 0; t < num_tensors; ++t) {
    if (total + numels[t] < total) return 0;   // sizes overflow
    total += numels[t];
  }
  const uint64_t chunk = opts->chunk_elems < total ? opts->chunk_elems : (total ? total : 1);
  const uint64_t nchunks = (total + chunk - 1) / chunk;
  const size_t ws = max_chunk_workspace(numels, num_tensors, total, chunk, leb);
  return staging_layout(chunk, ws, leb, opts->num_streams, nchunks).total;
}

size_t delta_pipeline_staging_bytes(const uint64_t* numels, int32_t num_tensors,
                                    const delta_pipeline_opts_t* opts) {
  return staging_bytes_impl(numels, num_tensors, opts, false);
}

size_t delta_pipeline_leb128_staging_bytes(const uint64_t* numels, int32_t num_tensors,
                                           const delta_pipeline_opts_t* opts) {
  return staging_bytes_impl(numels, num_tensors, opts, true);
}

}  // extern "C"

// Where the pipeline's output goes (pinned host memory).
struct PipeOut {
  bool leb;                  // indices gap + LEB128 coded, one segment per chunk
  int64_t* h_idx;            // plain: indices
  uint64_t h_idx_cap;
  uint8_t* h_bytes;          // coded: index bytes
  uint64_t h_bytes_cap;
  uint16_t* h_val;
  uint64_t h_val_cap;
  uint64_t* h_chunk_counts;  // coded: entries per chunk (host array)
  uint64_t h_num_chunks;
};

// Host-synchronous pipeline.  *h_count gets the entry total and, coded,
// *h_nbytes the byte total.
static delta_status_t pipeline_impl(const uint16_t* const* prevs, const uint16_t* const* nexts,
                                    const uint64_t* numels, int32_t T,
                                    const delta_pipeline_opts_t* opts, hipStream_t* streams,
                                    void* d_staging, size_t staging_bytes, const PipeOut& o,
                                    uint64_t* h_count, uint64_t* h_nbytes) {
  clear_error();
  if (!opts || opts->chunk_elems == 0 || opts->num_streams < 1 || opts->num_streams > 16) {
    set_error("bad pipeline options");
    return DELTA_ERR_INVALID_ARG;
  }
  if (T < 0 || (T > 0 && (!prevs || !nexts || !numels)) || !streams || !h_count ||
      (o.h_val_cap > 0 && !o.h_val) || (!o.leb && o.h_idx_cap > 0 && !o.h_idx) ||
      (o.leb && (!h_nbytes || (o.h_bytes_cap > 0 && !o.h_bytes)))) {
    set_error("NULL argument");
    return DELTA_ERR_INVALID_ARG;
  }
  uint64_t total = 0;
  for (int32_t t = 0; t < T; ++t) {
    if (numels[t] > 0 && (!prevs[t] || !nexts[t])) {
      set_error("tensor %d: NULL pointer", t);
      return DELTA_ERR_INVALID_ARG;
    }
    if (((uintptr_t)prevs[t] | (uintptr_t)nexts[t]) & 1u) {
      set_error("tensor %d: odd address", t);
      return DELTA_ERR_INVALID_ARG;
    }
    if (total + numels[t] < total) {
      set_error("total size overflows");
      return DELTA_ERR_INVALID_ARG;
    }
    total += numels[t];
  }
  if (total > 0 && total - 1 > 0x7FFFFFFFFFFFFFFFull) {
    set_error("total size exceeds int64");
    return DELTA_ERR_INDEX_OVERFLOW;
  }
  const int S = opts->num_streams;
  *h_count = 0;
  if (h_nbytes) *h_nbytes = 0;
  const uint64_t chunk = total == 0 ? 1 : (opts->chunk_elems < total ? opts->chunk_elems : total);
  const uint64_t nchunks = (total + chunk - 1) / chunk;
  if (o.leb && (o.h_num_chunks < nchunks || (nchunks > 0 && !o.h_chunk_counts))) {
    set_error("h_chunk_counts holds %llu entries, %llu chunks",
              (unsigned long long)o.h_num_chunks, (unsigned long long)nchunks);
    return DELTA_ERR_INVALID_ARG;
  }
  if (total == 0) return DELTA_OK;
  const size_t need = staging_bytes_impl(numels, T, opts, o.leb);
  if (!d_staging || (uintptr_t)d_staging % kAlign || staging_bytes < need) {
    set_error("staging: %zu bytes at %p, %zu needed (256-aligned)",
             staging_bytes, d_staging, need);
    return DELTA_ERR_WORKSPACE;
  }
  const size_t ws = max_chunk_workspace(numels, T, total, chunk, o.leb);
  const StagingLayout L = staging_layout(chunk, ws, o.leb, S, nchunks);
  const uint64_t bytes_cap = leb_bytes_per_entry(chunk) * chunk;

  // device views of the pinned host arrays (kernels store into them)
  DeliverArgs base;
  memset(&base, 0, sizeof(base));
  base.h_val_cap = o.h_val_cap;
  base.h_val = (uint16_t*)host_range_on_device(o.h_val, 2 * o.h_val_cap);
  bool pinned = o.h_val_cap == 0 || base.h_val;
  if (!o.leb) {
    base.h_idx_cap = o.h_idx_cap;
    base.h_idx = (int64_t*)host_range_on_device(o.h_idx, 8 * o.h_idx_cap);
    pinned = pinned && (o.h_idx_cap == 0 || base.h_idx);
  } else {
    base.h_bytes_cap = o.h_bytes_cap;
    base.h_bytes = (uint8_t*)host_range_on_device(o.h_bytes, o.h_bytes_cap);
    pinned = pinned && (o.h_bytes_cap == 0 || base.h_bytes);
  }
  if (!pinned) {
    set_error("host output arrays must be pinned host memory (hipHostMalloc / pin_memory)");
    return DELTA_ERR_INVALID_ARG;
  }
  if (base.h_val_cap && !base.h_val) base.h_val_cap = 0;
  if (base.h_idx_cap && !base.h_idx) base.h_idx_cap = 0;
  if (base.h_bytes_cap && !base.h_bytes) base.h_bytes_cap = 0;

  // Three roles: the reading stream runs every chunk's stage kernel (the
  // pass over the weights) back to back; the coding stream takes each
  // chunk's scan and finalize kernels as soon as its stage kernel is done,
  // while the next chunk is read; the delivery stream stores the chunks
  // into host memory in order.  With two streams reading and coding share
  // the first; with one, everything runs in order on it.
  const DeliverShape shape = o.leb ? kDeliverCoded : kDeliverPlain;
  hipStream_t const rs = streams[0];
  hipStream_t const cs = S > 2 ? streams[1] : streams[0];
  hipStream_t const ds = S > 2 ? streams[2] : streams[S - 1];
  // The events only order work on this device, so they skip the
  // system-scope fence (an L2 write-back on every record: about 20 us
  // between two kernels of the reading stream).  The host reads its
  // arrays after synchronising the streams.
  std::vector<hipEvent_t> staged(S, nullptr), extracted(S, nullptr), delivered(S, nullptr);
  const unsigned ev_flags = hipEventDisableTiming | hipEventDisableSystemFence;
  hipError_t e = hipSuccess;
  for (int i = 0; i < S && e == hipSuccess; ++i) {
    e = hipEventCreateWithFlags(&staged[i], ev_flags);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&extracted[i], ev_flags);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&delivered[i], ev_flags);
  }
  char* const stg = (char*)d_staging;
  uint64_t* const run = (uint64_t*)(stg + L.run);
  uint64_t* const d_chunk_counts = (uint64_t*)(stg + L.chunk_counts);
  if (e == hipSuccess) {
    hipLaunchKernelGGL(run_reset_kernel, dim3(1), dim3(64), 0, ds, run);
    e = hipGetLastError();
  }
  delta_status_t status = DELTA_OK;
  std::vector<SliceIn> sl;
  // Plain, with four or more slots, a delivery takes two consecutive
  // chunks (the second one's coding done covers the first's: the coding
  // stream runs in order): half the delivery kernels, each copying about
  // twice as much (Qwen3-14B: 29.8 against 30.1 ms).  Coded, pairs measured
  // slower (14.0 against 12.2-12.7 ms): its deliveries are short, and one
  // that waits for the next chunk holds the reading back through the slots.
  // With fewer slots the reading would wait on deliveries that wait on the
  // next chunk.
  const bool pair = S >= 4 && !o.leb;
  DeliverChunk pending = {};
  bool have_pending = false;
  uint64_t deliveries = 0;
  for (uint64_t c = 0; c < nchunks && e == hipSuccess; ++c) {
    const int slot = (int)(c % (uint64_t)S);
    char* stage = stg + L.per_stream * (size_t)slot;
    // The slot's previous chunk (c - S) must have been delivered before
    // chunk c is read into it.  With four or more slots the reading stream
    // waits only at every other chunk, on the delivery of chunk c - S + 1,
    // which covers the next chunk's slot too (deliveries run in order):
    // each wait is a packet the reading stream processes between two
    // stage kernels (Qwen3-14B coded: 13.0 against 13.5 ms).  With fewer
    // slots that would leave too little room between reading and delivery.
    const bool wait_every_other = S >= 4;
    if (c >= (uint64_t)S && ds != rs && (!wait_every_other || c % 2 == 0 || c == (uint64_t)S)) {
      const int after = wait_every_other ? (int)((c + 1) % (uint64_t)S) : slot;
      e = hipStreamWaitEvent(rs, delivered[after], 0);
      if (e != hipSuccess) break;
    }
    const uint64_t lo = c * chunk;
    const uint64_t hi = (total - lo < chunk) ? total : lo + chunk;
    chunk_slices(prevs, nexts, numels, T, lo, hi, sl);
    // coded: the chunk's positions as one gap + LEB128 segment based at
    // its first word, written by the extract itself
    const CodedOut co = {(uint8_t*)(stage + L.bytes), bytes_cap, (uint64_t*)(stage + L.nbytes),
                         (int64_t)lo, false, nullptr};
    const StageSplit split = {staged[slot], cs};
    const delta_status_t st =
        enqueue_extract(sl.data(), sl.size(), 0, true, stage + L.idx, (uint16_t*)(stage + L.val),
                        chunk, (uint64_t*)(stage + L.count), nullptr, stage + L.ws, L.ws_bytes, rs,
                        o.leb ? &co : nullptr, &split);
    if (st != DELTA_OK) {
      status = st;
      break;
    }
    const DeliverChunk cur = {o.leb ? nullptr : (const int64_t*)(stage + L.idx),
                              (const uint16_t*)(stage + L.val),
                              o.leb ? (const uint8_t*)(stage + L.bytes) : nullptr,
                              (const uint64_t*)(stage + L.count),
                              (const uint64_t*)(stage + L.nbytes)};
    if (pair && c % 2 == 0 && c + 1 < nchunks) {   // delivered with the next chunk
      pending = cur;
      have_pending = true;
      continue;
    }
    if (cs != ds) {
      e = hipEventRecord(extracted[slot], cs);
      if (e == hipSuccess) e = hipStreamWaitEvent(ds, extracted[slot], 0);
      if (e != hipSuccess) break;
    }
    DeliverArgs d = base;
    d.n = 0;
    if (have_pending) d.ch[d.n++] = pending;
    d.ch[d.n++] = cur;
    d.c = c + 1 - d.n;
    d.k = deliveries++;
    d.run = run;
    d.chunk_counts = o.leb ? d_chunk_counts : nullptr;
    d.xcds = shape.xcds;
    if (o.leb)
      hipLaunchKernelGGL((deliver_kernel<kCodedThreads, kCodedUnroll>),
                         dim3(kXcds * shape.per_xcd), dim3(kCodedThreads), 0, ds, d);
    else
      hipLaunchKernelGGL((deliver_kernel<kPlainThreads, kPlainUnroll>),
                         dim3(kXcds * shape.per_xcd), dim3(kPlainThreads), 0, ds, d);
    e = hipGetLastError();
    if (e == hipSuccess) e = hipEventRecord(delivered[slot], ds);
    if (e == hipSuccess && have_pending)
      e = hipEventRecord(delivered[(int)((c - 1) % (uint64_t)S)], ds);
    have_pending = false;
  }
  // Drain every stream whatever happened, so nothing is left in flight.
  for (int i = 0; i < S; ++i) {
    hipError_t e2 = hipStreamSynchronize(streams[i]);
    if (e == hipSuccess) e = e2;
  }
  uint64_t totals[2] = {0, 0};
  if (e == hipSuccess && status == DELTA_OK) {
    e = hipMemcpy(totals, run + 2 * (deliveries & 1), sizeof(totals), hipMemcpyDeviceToHost);
    if (e == hipSuccess && o.leb)
      e = hipMemcpy(o.h_chunk_counts, d_chunk_counts, sizeof(uint64_t) * nchunks,
                    hipMemcpyDeviceToHost);
  }
  for (int i = 0; i < S; ++i) {
    if (staged[i]) (void)hipEventDestroy(staged[i]);
    if (extracted[i]) (void)hipEventDestroy(extracted[i]);
    if (delivered[i]) (void)hipEventDestroy(delivered[i]);
  }
  if (e != hipSuccess) {
    set_error("HIP error in pipeline: %s", hipGetErrorString(e));
    return DELTA_ERR_HIP;
  }
  if (status != DELTA_OK) return status;   // a chunk could not be enqueued: no result
  const uint64_t entries = totals[0], nbytes = totals[1];
  *h_count = entries;
  if (h_nbytes) *h_nbytes = nbytes;
  const bool fits = entries <= o.h_val_cap && (o.leb ? nbytes <= o.h_bytes_cap
                                                     : entries <= o.h_idx_cap);
  if (!fits) {
    set_error("output has %llu entries (%llu index bytes); it does not fit",
             (unsigned long long)entries, (unsigned long long)nbytes);
    return DELTA_ERR_CAPACITY;
  }
  return DELTA_OK;
}

extern "C" delta_status_t delta_extract_pipelined(
    const uint16_t* const* prev_ptrs, const uint16_t* const* next_ptrs, const uint64_t* numels,
    int32_t num_tensors, const delta_pipeline_opts_t* opts, hipStream_t* streams,
    void* d_staging, size_t staging_bytes, int64_t* h_idx, uint16_t* h_val, uint64_t h_capacity,
    uint64_t* h_count) {
  PipeOut o;
  memset(&o, 0, sizeof(o));
  o.h_idx = h_idx;
  o.h_idx_cap = h_capacity;
  o.h_val = h_val;
  o.h_val_cap = h_capacity;
  return pipeline_impl(prev_ptrs, next_ptrs, numels, num_tensors, opts, streams, d_staging,
                       staging_bytes, o, h_count, nullptr);
}

extern "C" delta_status_t delta_extract_pipelined_leb128(
    const uint16_t* const* prev_ptrs, const uint16_t* const* next_ptrs, const uint64_t* numels,
    int32_t num_tensors, const delta_pipeline_opts_t* opts, hipStream_t* streams,
    void* d_staging, size_t staging_bytes, uint8_t* h_bytes, uint64_t h_bytes_capacity,
    uint16_t* h_val, uint64_t h_val_capacity, uint64_t* h_chunk_counts, uint64_t h_num_chunks,
    uint64_t* h_count, uint64_t* h_nbytes) {
  PipeOut o;
  memset(&o, 0, sizeof(o));
  o.leb = true;
  o.h_bytes = h_bytes;
  o.h_bytes_cap = h_bytes_capacity;
  o.h_val = h_val;
  o.h_val_cap = h_val_capacity;
  o.h_chunk_counts = h_chunk_counts;
  o.h_num_chunks = h_num_chunks;
  return pipeline_impl(prev_ptrs, next_ptrs, numels, num_tensors, opts, streams, d_staging,
                       staging_bytes, o, h_count, h_nbytes);
}
