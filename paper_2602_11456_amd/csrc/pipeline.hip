// Chunked extraction with the output streamed to pinned host memory
// (AuroraRL Sec. 5.2, "Overlapped extraction and transfer": the delta is cut
// into segments that are emitted as soon as each is encoded, striped
// round-robin over several parallel channels).
//
// The global index space of the tensor list is cut into chunks of
// `chunk_elems` words; a chunk may span several tensors and start inside
// one.  Chunk c runs on stream c mod S: its extract writes into that
// stream's device staging, then the chunk's count is copied to the host.
// The host takes chunks in order: it waits for chunk c's count, which fixes
// where chunk c's entries land in the host arrays, and enqueues the copy of
// chunk c's (idx, val) behind it on the same stream, before it enqueues
// chunk c + S there (so the staging is never overwritten early).  Up to S
// chunks are in flight: extracts on some streams overlap device-to-host
// copies on the others.
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
      out.push_back({prevs[t] + (a - base), nexts[t] + (a - base), b - a, a, (uint32_t)t});
    base += n;
  }
}


struct StagingLayout {
  size_t idx, val, count, ws, ws_bytes, per_stream;
};

StagingLayout staging_layout(uint64_t chunk, size_t ws_bytes) {
  StagingLayout L;
  L.idx = 0;
  L.val = align_up(L.idx + 8 * chunk);
  L.count = align_up(L.val + 2 * chunk);
  L.ws = align_up(L.count + 8);
  L.ws_bytes = ws_bytes;
  L.per_stream = align_up(L.ws + ws_bytes);
  return L;
}

// Largest workspace any chunk's extract needs (tiles at worst alignment).
size_t max_chunk_workspace(const uint64_t* numels, int32_t T, uint64_t total, uint64_t chunk) {
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
    const size_t need = workspace_bytes(tiles, rows, kDefaultStageCap);
    if (need > best) best = need;
  }
  return best;
}

}  // namespace

extern "C" {

size_t delta_pipeline_staging_bytes(const uint64_t* numels, int32_t num_tensors,
                                    const delta_pipeline_opts_t* opts) {
  if (!opts || opts->chunk_elems == 0 || opts->num_streams < 1 || opts->num_streams > 16 ||
      num_tensors < 0 || (num_tensors > 0 && !numels))
    return 0;
  uint64_t total = 0;
  for (int32_t t = 0; t < num_tensors; ++t) total += numels[t];
  const uint64_t chunk = opts->chunk_elems < total ? opts->chunk_elems : (total ? total : 1);
  const size_t ws = max_chunk_workspace(numels, num_tensors, total, chunk);
  return staging_layout(chunk, ws).per_stream * (size_t)opts->num_streams;
}

}  // extern "C"

// Host-synchronous pipeline.  Defined with C linkage below.
static delta_status_t pipeline_impl(const uint16_t* const* prevs, const uint16_t* const* nexts,
                                    const uint64_t* numels, int32_t T,
                                    const delta_pipeline_opts_t* opts, hipStream_t* streams,
                                    void* d_staging, size_t staging_bytes, int64_t* h_idx,
                                    uint16_t* h_val, uint64_t h_cap, uint64_t* h_count) {
  clear_error();
  if (!opts || opts->chunk_elems == 0 || opts->num_streams < 1 || opts->num_streams > 16) {
    set_error("bad pipeline options");
    return DELTA_ERR_INVALID_ARG;
  }
  if (T < 0 || (T > 0 && (!prevs || !nexts || !numels)) || !streams || !h_count ||
      (h_cap > 0 && (!h_idx || !h_val))) {
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
    total += numels[t];
  }
  const int S = opts->num_streams;
  *h_count = 0;
  if (total == 0) return DELTA_OK;
  const uint64_t chunk = opts->chunk_elems < total ? opts->chunk_elems : total;
  const size_t need = delta_pipeline_staging_bytes(numels, T, opts);
  if (!d_staging || (uintptr_t)d_staging % kAlign || staging_bytes < need) {
    set_error("staging: %zu bytes at %p, %zu needed (256-aligned)",
             staging_bytes, d_staging, need);
    return DELTA_ERR_WORKSPACE;
  }
  const size_t ws = max_chunk_workspace(numels, T, total, chunk);
  const StagingLayout L = staging_layout(chunk, ws);
  const uint64_t nchunks = (total + chunk - 1) / chunk;

  uint64_t* h_counts = nullptr;   // per-chunk counts land here (pinned)
  hipError_t e = hipHostMalloc((void**)&h_counts, sizeof(uint64_t) * nchunks, hipHostMallocDefault);
  if (e != hipSuccess) {
    set_error("hipHostMalloc: %s", hipGetErrorString(e));
    return DELTA_ERR_HIP;
  }

  std::vector<SliceIn> sl;
  uint64_t offset = 0;   // host position of the next chunk's first entry
  uint64_t finished = 0; // chunks whose data copy is enqueued
  uint64_t issued = 0;   // chunks whose extract and count copy are enqueued
  delta_status_t status = DELTA_OK;

  auto stage_of = [&](uint64_t c) { return (char*)d_staging + L.per_stream * (c % S); };
  auto finish = [&](uint64_t c) -> hipError_t {
    hipStream_t st = streams[c % S];
    hipError_t err = hipStreamSynchronize(st);
    if (err != hipSuccess) return err;
    const uint64_t cnt = h_counts[c];
    char* stage = stage_of(c);
    if (offset < h_cap && cnt > 0) {
      const uint64_t m = (h_cap - offset < cnt) ? h_cap - offset : cnt;
      err = hipMemcpyAsync(h_idx + offset, stage + L.idx, 8 * m, hipMemcpyDeviceToHost, st);
      if (err != hipSuccess) return err;
      err = hipMemcpyAsync(h_val + offset, stage + L.val, 2 * m, hipMemcpyDeviceToHost, st);
      if (err != hipSuccess) return err;
    }
    offset += cnt;
    finished = c + 1;
    return hipSuccess;
  };

  for (uint64_t c = 0; c < nchunks && e == hipSuccess; ++c) {
    if (c >= (uint64_t)S) {
      e = finish(c - S);
      if (e != hipSuccess) break;
    }
    const uint64_t lo = c * chunk;
    const uint64_t hi = (total - lo < chunk) ? total : lo + chunk;
    chunk_slices(prevs, nexts, numels, T, lo, hi, sl);
    char* stage = stage_of(c);
    const delta_status_t st =
        enqueue_extract(sl.data(), sl.size(), 0, true, stage + L.idx, (uint16_t*)(stage + L.val),
                        chunk, (uint64_t*)(stage + L.count), nullptr, stage + L.ws, L.ws_bytes,
                        streams[c % S]);
    if (st != DELTA_OK) {
      status = st;
      break;
    }
    e = hipMemcpyAsync(&h_counts[c], stage + L.count, 8, hipMemcpyDeviceToHost, streams[c % S]);
    if (e == hipSuccess) issued = c + 1;
  }
  while (e == hipSuccess && status == DELTA_OK && finished < issued) e = finish(finished);
  // Drain every stream whatever happened, so no copy is left in flight.
  for (int s = 0; s < S; ++s) {
    hipError_t e2 = hipStreamSynchronize(streams[s]);
    if (e == hipSuccess) e = e2;
  }
  (void)hipHostFree(h_counts);
  if (e != hipSuccess) {
    set_error("HIP error in pipeline: %s", hipGetErrorString(e));
    *h_count = 0;
    return DELTA_ERR_HIP;
  }
  if (status != DELTA_OK) {   // a chunk could not be enqueued: no partial result
    *h_count = 0;
    return status;
  }
  *h_count = offset;
  if (offset > h_cap) {
    set_error("output has %llu entries, capacity %llu",
             (unsigned long long)offset, (unsigned long long)h_cap);
    status = DELTA_ERR_CAPACITY;
  }
  return status;
}

extern "C" delta_status_t delta_extract_pipelined(
    const uint16_t* const* prev_ptrs, const uint16_t* const* next_ptrs, const uint64_t* numels,
    int32_t num_tensors, const delta_pipeline_opts_t* opts, hipStream_t* streams,
    void* d_staging, size_t staging_bytes, int64_t* h_idx, uint16_t* h_val, uint64_t h_capacity,
    uint64_t* h_count) {
  return pipeline_impl(prev_ptrs, next_ptrs, numels, num_tensors, opts, streams, d_staging,
                       staging_bytes, h_idx, h_val, h_capacity, h_count);
}
