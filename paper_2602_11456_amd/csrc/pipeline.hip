// Chunked extraction with the output streamed to pinned host memory
// (AuroraRL Sec. 5.2, "Overlapped extraction and transfer": the delta is cut
// into segments that are emitted as soon as each is encoded, striped
// round-robin over several parallel channels).
//
// The global index space of the tensor list is cut into chunks of
// `chunk_elems` words; a chunk may span several tensors and start inside
// one.  Chunk c is extracted on stream c mod S into that stream's device
// staging (coded: its indices are then gap + LEB128 coded there), and its
// count is copied to the host.  The host takes chunks in order: it waits
// for chunk c's count, which fixes where chunk c's entries land in the host
// arrays, and enqueues the copies of chunk c on one copy stream of the
// library's own (device-to-host copies from several streams at once share
// the host link less well than back-to-back copies from one).  The extract
// of chunk c + S waits on an event recorded after those copies, so the
// staging is never overwritten early.  Up to S chunks are in flight:
// extracts on the compute streams overlap the copies.
#include <string.h>

#include <vector>

#include "aurora_delta.h"
#include "delta_internal.h"
#include "leb128.h"

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
  size_t idx, val, count, nbytes, bytes, enc_ws, ws, ws_bytes, per_stream;
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

StagingLayout staging_layout(uint64_t chunk, size_t ws_bytes, bool leb) {
  StagingLayout L;
  L.idx = 0;
  L.val = align_up(L.idx + 8 * chunk);
  L.count = align_up(L.val + 2 * chunk);
  L.nbytes = L.count + 8;
  L.bytes = align_up(L.nbytes + 8);
  L.enc_ws = align_up(L.bytes + (leb ? leb_bytes_per_entry(chunk) * chunk : 0));
  L.ws = align_up(L.enc_ws + (leb ? enc_layout(chunk).total : 0));
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

static size_t staging_bytes_impl(const uint64_t* numels, int32_t num_tensors,
                                 const delta_pipeline_opts_t* opts, bool leb) {
  if (!opts || opts->chunk_elems == 0 || opts->num_streams < 1 || opts->num_streams > 16 ||
      num_tensors < 0 || (num_tensors > 0 && !numels))
    return 0;
  uint64_t total = 0;
  for (int32_t t = 0; t < num_tensors; ++t) total += numels[t];
  const uint64_t chunk = opts->chunk_elems < total ? opts->chunk_elems : (total ? total : 1);
  const size_t ws = max_chunk_workspace(numels, num_tensors, total, chunk);
  return staging_layout(chunk, ws, leb).per_stream * (size_t)opts->num_streams;
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
    total += numels[t];
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
  const size_t ws = max_chunk_workspace(numels, T, total, chunk);
  const StagingLayout L = staging_layout(chunk, ws, o.leb);
  const uint64_t bytes_cap = leb_bytes_per_entry(chunk) * chunk;

  // per chunk: entry count and (coded) byte count land here (pinned)
  uint64_t* h_counts = nullptr;
  hipError_t e =
      hipHostMalloc((void**)&h_counts, sizeof(uint64_t) * 2 * nchunks, hipHostMallocDefault);
  if (e != hipSuccess) {
    set_error("hipHostMalloc: %s", hipGetErrorString(e));
    return DELTA_ERR_HIP;
  }

  hipStream_t cs = nullptr;   // carries every data copy
  std::vector<hipEvent_t> copied(S, nullptr);   // per staging slot: its last copies are done
  e = hipStreamCreateWithFlags(&cs, hipStreamNonBlocking);
  for (int i = 0; i < S && e == hipSuccess; ++i)
    e = hipEventCreateWithFlags(&copied[i], hipEventDisableTiming);

  std::vector<SliceIn> sl;
  uint64_t offset = 0;   // host position of the next chunk's first entry
  uint64_t boffset = 0;  // coded: host position of the next chunk's first byte
  uint64_t finished = 0; // chunks whose data copies are enqueued
  uint64_t issued = 0;   // chunks whose extract and count copy are enqueued
  delta_status_t status = DELTA_OK;

  auto stage_of = [&](uint64_t c) { return (char*)d_staging + L.per_stream * (c % S); };
  auto copy_out = [&](void* dst, const void* src, uint64_t pos, uint64_t cap, uint64_t n,
                      size_t elem, hipStream_t st) -> hipError_t {
    if (pos >= cap || n == 0) return hipSuccess;
    const uint64_t m = (cap - pos < n) ? cap - pos : n;
    return hipMemcpyAsync((char*)dst + elem * pos, src, elem * m, hipMemcpyDeviceToHost, st);
  };
  auto finish = [&](uint64_t c) -> hipError_t {
    hipError_t err = hipStreamSynchronize(streams[c % S]);
    if (err != hipSuccess) return err;
    hipStream_t st = cs;
    const uint64_t cnt = h_counts[2 * c];
    char* stage = stage_of(c);
    if (!o.leb) {
      err = copy_out(o.h_idx, stage + L.idx, offset, o.h_idx_cap, cnt, 8, st);
    } else {
      o.h_chunk_counts[c] = cnt;
      const uint64_t nb = h_counts[2 * c + 1];
      err = copy_out(o.h_bytes, stage + L.bytes, boffset, o.h_bytes_cap, nb, 1, st);
      boffset += nb;
    }
    if (err == hipSuccess) err = copy_out(o.h_val, stage + L.val, offset, o.h_val_cap, cnt, 2, st);
    if (err == hipSuccess) err = hipEventRecord(copied[c % S], st);
    offset += cnt;
    finished = c + 1;
    return err;
  };
  // Coded: the chunk's indices as one segment based at its first word; the
  // encoder reads the entry count that the extract left in device memory.
  const EncLayout E = enc_layout(chunk);
  auto enqueue_encode = [&](uint64_t c) -> hipError_t {
    char* stage = stage_of(c);
    EncArgs a;
    memset(&a, 0, sizeof(a));
    a.idx = (const int64_t*)(stage + L.idx);
    a.count = chunk;
    a.d_count_in = (const uint64_t*)(stage + L.count);
    a.segs = {nullptr, nullptr, 0, (int64_t)(c * chunk)};
    a.out = (uint8_t*)(stage + L.bytes);
    a.capacity = bytes_cap;
    a.d_nbytes = (uint64_t*)(stage + L.nbytes);
    a.tile_bytes = (uint32_t*)(stage + L.enc_ws + E.tile_bytes);
    return launch_leb128_encode(a, (uint64_t*)(stage + L.enc_ws + E.group_sum),
                                (uint64_t*)(stage + L.enc_ws + E.group_excl), streams[c % S]);
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
    if (c >= (uint64_t)S) {   // the slot's previous chunk must have left it
      e = hipStreamWaitEvent(streams[c % S], copied[c % S], 0);
      if (e != hipSuccess) break;
    }
    const delta_status_t st =
        enqueue_extract(sl.data(), sl.size(), 0, true, stage + L.idx, (uint16_t*)(stage + L.val),
                        chunk, (uint64_t*)(stage + L.count), nullptr, stage + L.ws, L.ws_bytes,
                        streams[c % S]);
    if (st != DELTA_OK) {
      status = st;
      break;
    }
    if (o.leb) e = enqueue_encode(c);
    // the count (and, coded, the byte count right after it) to the host
    if (e == hipSuccess)
      e = hipMemcpyAsync(&h_counts[2 * c], stage + L.count, o.leb ? 16 : 8,
                         hipMemcpyDeviceToHost, streams[c % S]);
    if (e == hipSuccess) issued = c + 1;
  }
  while (e == hipSuccess && status == DELTA_OK && finished < issued) e = finish(finished);
  // Drain every stream whatever happened, so no copy is left in flight.
  for (int s = 0; s < S; ++s) {
    hipError_t e2 = hipStreamSynchronize(streams[s]);
    if (e == hipSuccess) e = e2;
  }
  if (cs) {
    hipError_t e2 = hipStreamSynchronize(cs);
    if (e == hipSuccess) e = e2;
    (void)hipStreamDestroy(cs);
  }
  for (hipEvent_t ev : copied)
    if (ev) (void)hipEventDestroy(ev);
  (void)hipHostFree(h_counts);
  if (e != hipSuccess) {
    set_error("HIP error in pipeline: %s", hipGetErrorString(e));
    return DELTA_ERR_HIP;
  }
  if (status != DELTA_OK) return status;   // a chunk could not be enqueued: no result
  *h_count = offset;
  if (h_nbytes) *h_nbytes = boffset;
  const bool fits = offset <= o.h_val_cap && (o.leb ? boffset <= o.h_bytes_cap
                                                    : offset <= o.h_idx_cap);
  if (!fits) {
    set_error("output has %llu entries (%llu index bytes); it does not fit",
             (unsigned long long)offset, (unsigned long long)boffset);
    status = DELTA_ERR_CAPACITY;
  }
  return status;
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
