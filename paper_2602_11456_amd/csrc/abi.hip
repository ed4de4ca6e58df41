// C ABI entry points: argument validation, workspace carving, tensor tables
// and launch order.  Every computation runs in the kernels of extract.hip
// and apply.hip; this file only prepares and enqueues them.
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "aurora_delta.h"
#include "delta_internal.h"
#include "leb128.h"
#include "hash.h"

using namespace aurora;

static thread_local std::string g_last_error;

namespace aurora {

void set_error(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
}

void clear_error() { g_last_error.clear(); }

static hipEvent_t g_scan_events[2] = {nullptr, nullptr};

hipError_t record_scan_event(int which, hipStream_t stream) {
  const hipEvent_t ev = g_scan_events[which];
  return ev ? hipEventRecord(ev, stream) : hipSuccess;
}

}  // namespace aurora

namespace {

delta_status_t fail(delta_status_t s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
delta_status_t fail(delta_status_t s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

delta_status_t ok() {
  g_last_error.clear();
  return DELTA_OK;
}

delta_status_t hip_fail(hipError_t e, const char* what) {
  return fail(DELTA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool odd(const void* p) { return ((uintptr_t)p & 1u) != 0; }

// Descriptor table of the non-empty slices: tile ranges, alignment, and the
// tensor_offsets slots each slice's first tile writes.  Returns the number
// of tiles.
uint64_t build_descs(const SliceIn* slices, size_t num_slices, std::vector<TensorDesc>& out) {
  out.clear();
  uint64_t tiles = 0;
  uint32_t next_slot = 0;   // first tensor_offsets slot not yet owned
  for (size_t i = 0; i < num_slices; ++i) {
    const SliceIn& s = slices[i];
    if (s.n == 0) continue;
    TensorDesc d;
    memset(&d, 0, sizeof(d));
    d.prev = s.prev;
    d.next = s.next;
    d.n = s.n;
    d.base = s.base;
    d.first_tile = tiles;
    const uint32_t hp = head_words(s.prev), hq = head_words(s.next);
    d.vec = (hp == hq) ? 1u : 0u;
    d.head = d.vec ? hp : 0u;
    d.off_lo = next_slot;
    d.slot = s.tensor;
    d.seg_base = s.seg_base;
    next_slot = s.tensor + 1;
    tiles += tiles_for(d.n, d.head);
    out.push_back(d);
  }
  return tiles;
}

size_t multi_workspace_bound(const uint64_t* numels, int32_t T, bool coded = false) {
  uint64_t tiles = 0;
  for (int32_t t = 0; t < T; ++t) tiles += tiles_bound(numels[t]);
  return workspace_bytes(tiles, (uint64_t)(T > 0 ? T : 0), kDefaultStageCap, coded);
}

// The slices of a tensor list (one per tensor, word 0 of tensor t at the
// sum of the sizes before it), after the checks every list entry point
// shares.
delta_status_t list_slices(const uint16_t* const* prev_ptrs, const uint16_t* const* next_ptrs,
                           const uint64_t* numels, int32_t num_tensors,
                           std::vector<SliceIn>& slices) {
  if (num_tensors < 0) return fail(DELTA_ERR_INVALID_ARG, "num_tensors < 0");
  if (num_tensors > 0 && (!prev_ptrs || !next_ptrs || !numels))
    return fail(DELTA_ERR_INVALID_ARG, "tensor arrays are NULL");
  slices.clear();
  slices.reserve(num_tensors);
  uint64_t base = 0;
  for (int32_t t = 0; t < num_tensors; ++t) {
    if (numels[t] > 0 && (!prev_ptrs[t] || !next_ptrs[t]))
      return fail(DELTA_ERR_INVALID_ARG, "tensor %d: NULL pointer", t);
    if (odd(prev_ptrs[t]) || odd(next_ptrs[t]))
      return fail(DELTA_ERR_INVALID_ARG, "tensor %d: not 2-byte aligned", t);
    if (base + numels[t] < base) return fail(DELTA_ERR_INVALID_ARG, "total size overflows");
    slices.push_back({prev_ptrs[t], next_ptrs[t], numels[t], base, (uint32_t)t, base});
    base += numels[t];
  }
  if (base > 0 && base - 1 > 0x7FFFFFFFFFFFFFFFull)
    return fail(DELTA_ERR_INDEX_OVERFLOW, "total size exceeds int64");
  return DELTA_OK;
}

delta_status_t check_workspace(void* ws, size_t have, size_t need) {
  if (need == 0) return DELTA_OK;
  if (!ws) return fail(DELTA_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if ((uintptr_t)ws % kAlign)
    return fail(DELTA_ERR_WORKSPACE, "workspace must be %zu-byte aligned", kAlign);
  if (have < need)
    return fail(DELTA_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", have, need);
  return DELTA_OK;
}

}  // namespace

namespace aurora {

delta_status_t enqueue_extract(const SliceIn* slices, size_t num_slices, uint32_t num_tensors,
                               bool idx64, void* out_idx, uint16_t* out_val, uint64_t capacity,
                               uint64_t* d_count, uint64_t* d_offsets, void* workspace,
                               size_t have, hipStream_t stream, const CodedOut* coded,
                               const StageSplit* split, bool count_only,
                               const PreparedTable* prepared) {
  if (count_only) {
    coded = nullptr;
    split = nullptr;
    d_offsets = nullptr;
  }
  std::vector<TensorDesc> built;
  const uint64_t tiles = prepared ? prepared->tiles : build_descs(slices, num_slices, built);
  const std::vector<TensorDesc>& descs = prepared ? prepared->descs : built;
  if (tiles > 0xFFFFFFFFull / kThreads)
    return fail(DELTA_ERR_INVALID_ARG, "too many words for one launch (%llu tiles)",
                (unsigned long long)tiles);
  if (coded && !coded->per_tensor) d_offsets = nullptr;
  uint64_t* d_byte_offsets = (coded && coded->per_tensor) ? coded->d_byte_offsets : nullptr;
  if (tiles == 0) {
    hipError_t e = launch_reset(d_count, d_offsets, d_offsets ? num_tensors + 1 : 0, stream);
    if (e == hipSuccess && coded)
      e = launch_reset(coded->d_nbytes, d_byte_offsets, d_byte_offsets ? num_tensors + 1 : 0,
                       stream);
    if (e == hipSuccess && split) {
      e = hipEventRecord(split->staged, stream);
      if (e == hipSuccess && split->rest != stream) e = hipStreamWaitEvent(split->rest, split->staged, 0);
    }
    if (e != hipSuccess) return hip_fail(e, "reset launch");
    return ok();
  }
  const bool cd = coded != nullptr;
  const uint32_t cap = stage_cap_for(have, tiles, descs.size(), cd);
  if (cap == 0 || !workspace || (uintptr_t)workspace % kAlign)
    return fail(DELTA_ERR_WORKSPACE, "workspace: %zu bytes at %p; at least %zu bytes, %zu-aligned",
                have, workspace, workspace_bytes(tiles, descs.size(), kMinStageCap, cd), kAlign);
  const WorkspaceLayout L = workspace_layout(tiles, descs.size(), cd);
  char* ws = (char*)workspace;
  ExtractArgs a;
  memset(&a, 0, sizeof(a));
  a.num_tiles = tiles;
  a.num_tensors = num_tensors;
  a.stage_cap = cap;
  a.stage_stride = cap + kSlotPad;
  a.out_idx = out_idx;
  a.out_val = out_val;
  a.capacity = capacity;
  a.d_count = d_count;
  a.d_tensor_offsets = d_offsets;
  a.counts = (uint32_t*)(ws + L.counts);
  a.group_sum = (uint64_t*)(ws + L.group_sum);
  a.group_excl = (uint64_t*)(ws + L.group_excl);
  a.stage = (uint32_t*)(ws + L.stage);
  hipError_t e;
  if (descs.size() > (size_t)kInlineDescs && prepared) {
    a.table = prepared->d_table;
    a.tile_map = prepared->d_map;
  } else if (descs.size() > (size_t)kInlineDescs) {
    TensorDesc* table = (TensorDesc*)(ws + L.table);
    uint32_t* map = (uint32_t*)(ws + L.map);
    e = launch_upload_words((const uint64_t*)descs.data(), descs.size() * sizeof(TensorDesc) / 8,
                            (uint64_t*)table, stream);
    if (e != hipSuccess) return hip_fail(e, "table upload launch");
    e = launch_build_tile_map(table, (uint32_t)descs.size(), map, stream);
    if (e != hipSuccess) return hip_fail(e, "tile map launch");
    a.table = table;
    a.tile_map = map;
  } else {
    for (size_t i = 0; i < descs.size(); ++i) a.inl[i] = descs[i];
    a.num_inline = (uint32_t)descs.size();
  }
  bool all_vec = true;
  for (const TensorDesc& t : descs) all_vec = all_vec && t.vec;
  if (count_only) {
    e = launch_count(a, all_vec, stream);
  } else if (coded) {
    a.tile_rec = (uint64_t*)(ws + L.tile_rec);
    a.group_bexcl = (uint64_t*)(ws + L.group_bexcl);
    a.group_prev = (int64_t*)(ws + L.group_prev);
    a.code_out = coded->out;
    a.code_capacity = coded->capacity;
    a.d_nbytes = coded->d_nbytes;
    a.code_base = coded->per_tensor ? 0 : coded->base;
    a.seg_per_tensor = coded->per_tensor ? 1u : 0u;
    a.group_first_local = (int64_t*)(ws + L.group_first_local);
    a.d_tensor_byte_offsets = d_byte_offsets;
    e = launch_extract_coded(a, all_vec, stream, split);
  } else {
    e = launch_extract(a, idx64, all_vec, stream, split);
  }
  if (e != hipSuccess) return hip_fail(e, "extract launch");
  return ok();
}

}  // namespace aurora

extern "C" {

int delta_abi_version(void) { return AURORA_DELTA_ABI_VERSION; }

const char* delta_status_string(int status) {
  switch (status) {
    case DELTA_OK: return "DELTA_OK";
    case DELTA_ERR_INVALID_ARG: return "DELTA_ERR_INVALID_ARG";
    case DELTA_ERR_INDEX_OVERFLOW: return "DELTA_ERR_INDEX_OVERFLOW";
    case DELTA_ERR_CAPACITY: return "DELTA_ERR_CAPACITY";
    case DELTA_ERR_OUT_OF_RANGE: return "DELTA_ERR_OUT_OF_RANGE";
    case DELTA_ERR_VERSION: return "DELTA_ERR_VERSION";
    case DELTA_ERR_WORKSPACE: return "DELTA_ERR_WORKSPACE";
    case DELTA_ERR_HIP: return "DELTA_ERR_HIP";
    case DELTA_ERR_INTEGRITY: return "DELTA_ERR_INTEGRITY";
    default: return "DELTA_ERR_UNKNOWN";
  }
}

const char* delta_last_error(void) { return g_last_error.c_str(); }

delta_status_t delta_set_scan_events(hipEvent_t before, hipEvent_t after) {
  if ((before == nullptr) != (after == nullptr))
    return fail(DELTA_ERR_INVALID_ARG, "set both scan events or neither");
  g_scan_events[0] = before;
  g_scan_events[1] = after;
  return ok();
}

size_t delta_extract_workspace_bytes(uint64_t numel) {
  return workspace_bytes(tiles_bound(numel), 1, kDefaultStageCap);
}

size_t delta_extract_multi_workspace_bytes(const uint64_t* numels, int32_t num_tensors) {
  if (num_tensors < 0 || (num_tensors > 0 && !numels)) return 0;
  return multi_workspace_bound(numels, num_tensors);
}

size_t delta_apply_multi_workspace_bytes(int32_t num_tensors) {
  if (num_tensors < 0) return 0;
  return align_up(8 * ((size_t)num_tensors + 1)) + align_up(8 * (size_t)num_tensors);
}

size_t delta_apply_multi_sorted_workspace_bytes(int32_t num_tensors) {
  if (num_tensors < 0) return 0;
  return delta_apply_multi_workspace_bytes(num_tensors) + align_up(8 * ((size_t)num_tensors + 1));
}

}  // extern "C"

// Argument checks of delta_extract and delta_extract_noalloc (no HIP call).
static delta_status_t check_extract_args(const uint16_t* prev, const uint16_t* next,
                                         uint64_t numel, delta_index_t index_type,
                                         void* out_idx, uint16_t* out_val, uint64_t capacity,
                                         uint64_t* d_count) {
  if (index_type != DELTA_INDEX_I32 && index_type != DELTA_INDEX_I64)
    return fail(DELTA_ERR_INVALID_ARG, "unknown index type %d", (int)index_type);
  if (!d_count) return fail(DELTA_ERR_INVALID_ARG, "d_count is NULL");
  if (numel > 0 && (!prev || !next)) return fail(DELTA_ERR_INVALID_ARG, "prev/next is NULL");
  if (odd(prev) || odd(next)) return fail(DELTA_ERR_INVALID_ARG, "prev/next not 2-byte aligned");
  if (capacity > 0 && (!out_idx || !out_val))
    return fail(DELTA_ERR_INVALID_ARG, "out_idx/out_val is NULL with capacity %llu",
                (unsigned long long)capacity);
  if ((uintptr_t)out_idx % (index_type == DELTA_INDEX_I64 ? 8 : 4) || odd(out_val))
    return fail(DELTA_ERR_INVALID_ARG, "out_idx/out_val not aligned to their element size");
  if (index_type == DELTA_INDEX_I32 && numel > 0 && numel - 1 > 0x7FFFFFFFull)
    return fail(DELTA_ERR_INDEX_OVERFLOW, "numel %llu needs int64 indices",
                (unsigned long long)numel);
  return DELTA_OK;
}

extern "C" {

delta_status_t delta_extract(const uint16_t* prev, const uint16_t* next, uint64_t numel,
                             delta_index_t index_type, void* out_idx, uint16_t* out_val,
                             uint64_t capacity, uint64_t* d_count, void* workspace,
                             size_t workspace_bytes, hipStream_t stream) {
  const delta_status_t s =
      check_extract_args(prev, next, numel, index_type, out_idx, out_val, capacity, d_count);
  if (s != DELTA_OK) return s;
  const SliceIn slice{prev, next, numel, 0, 0, 0};
  return enqueue_extract(&slice, 1, 1, index_type == DELTA_INDEX_I64, out_idx, out_val, capacity,
                         d_count, nullptr, workspace, workspace_bytes, stream);
}

}  // extern "C"

// ----------------------------------------------- extract without allocation
//
// delta_extract_noalloc keeps its scratch (tile counts, group sums, staging
// slots) in this file-scope device array instead of a caller workspace.
// Every GPU the library runs on holds its own copy, at its own address,
// until the process ends.  Host code never passes `noalloc_scratch` itself
// to a kernel (in host code the name is only a stand-in for the symbol):
// the device address comes from hipGetSymbolAddress, resolved once per
// device with that device current, and kept in g_noalloc_ptr.  Nothing in
// the array has to start at zero: the extract writes every tile count and
// group sum it later reads.
static __device__ __align__(256) unsigned char noalloc_scratch[DELTA_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_noalloc_mu;
void* g_noalloc_ptr[kMaxDevices] = {};

// Device address of `noalloc_scratch` on the device that runs `stream`.
delta_status_t noalloc_scratch_for(hipStream_t stream, void** out) {
  int dev = -1;
  hipError_t e = stream ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "device of the stream");
  if (dev < 0 || dev >= kMaxDevices) return fail(DELTA_ERR_HIP, "device %d out of range", dev);
  std::lock_guard<std::mutex> lock(g_noalloc_mu);
  if (!g_noalloc_ptr[dev]) {
    int cur = -1;
    e = hipGetDevice(&cur);
    if (e == hipSuccess && cur != dev) e = hipSetDevice(dev);
    if (e != hipSuccess) return hip_fail(e, "select the stream's device");
    void* p = nullptr;
    const hipError_t es = hipGetSymbolAddress(&p, HIP_SYMBOL(noalloc_scratch));
    if (cur != dev) e = hipSetDevice(cur);
    if (es != hipSuccess) return hip_fail(es, "hipGetSymbolAddress(noalloc_scratch)");
    if (e != hipSuccess) return hip_fail(e, "restore the current device");
    if (!p || (uintptr_t)p % kAlign)
      return fail(DELTA_ERR_HIP, "scratch array at %p is not %zu-byte aligned", p, kAlign);
    g_noalloc_ptr[dev] = p;
  }
  *out = g_noalloc_ptr[dev];
  return DELTA_OK;
}

}  // namespace

extern "C" {

delta_status_t delta_extract_noalloc(const uint16_t* prev, const uint16_t* next, uint64_t numel,
                                     delta_index_t index_type, void* out_idx, uint16_t* out_val,
                                     uint64_t capacity, uint64_t* d_count, hipStream_t stream) {
  delta_status_t s =
      check_extract_args(prev, next, numel, index_type, out_idx, out_val, capacity, d_count);
  if (s != DELTA_OK) return s;
  if (numel > DELTA_NOALLOC_MAX_WORDS)
    return fail(DELTA_ERR_WORKSPACE,
                "delta_extract_noalloc: numel %llu exceeds its maximum of %llu words (use "
                "delta_extract with a workspace)",
                (unsigned long long)numel, (unsigned long long)DELTA_NOALLOC_MAX_WORDS);
  void* ws = nullptr;
  if (numel > 0) {
    s = noalloc_scratch_for(stream, &ws);
    if (s != DELTA_OK) return s;
  }
  const SliceIn slice{prev, next, numel, 0, 0, 0};
  return enqueue_extract(&slice, 1, 1, index_type == DELTA_INDEX_I64, out_idx, out_val, capacity,
                         d_count, nullptr, ws, numel > 0 ? (size_t)DELTA_NOALLOC_SCRATCH_BYTES : 0,
                         stream);
}

delta_status_t delta_extract_multi(const uint16_t* const* prev_ptrs,
                                   const uint16_t* const* next_ptrs, const uint64_t* numels,
                                   int32_t num_tensors, int64_t* out_idx, uint16_t* out_val,
                                   uint64_t capacity, uint64_t* d_count,
                                   uint64_t* d_tensor_offsets, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream) {
  if (!d_count) return fail(DELTA_ERR_INVALID_ARG, "d_count is NULL");
  if (capacity > 0 && (!out_idx || !out_val))
    return fail(DELTA_ERR_INVALID_ARG, "out_idx/out_val is NULL with capacity %llu",
                (unsigned long long)capacity);
  if ((uintptr_t)out_idx % 8 || odd(out_val))
    return fail(DELTA_ERR_INVALID_ARG, "out_idx/out_val not aligned to their element size");
  std::vector<SliceIn> slices;
  const delta_status_t st = list_slices(prev_ptrs, next_ptrs, numels, num_tensors, slices);
  if (st != DELTA_OK) return st;
  return enqueue_extract(slices.data(), slices.size(), (uint32_t)num_tensors, true, out_idx,
                         out_val, capacity, d_count, d_tensor_offsets, workspace,
                         workspace_bytes, stream);
}

}  // extern "C"

// --------------------------------------------------------- tensor-list plan
//
// The slice descriptors of a tensor list, and past kInlineDescs of them the
// device table and tile map, built once: a training loop extracts the same
// tensors (the same pointers) every step, and the per-call upload (ten
// small launches and the tile map for 399 tensors, ~45 us) then goes away.
struct delta_multi_plan {
  int device;
  int32_t num_tensors;
  size_t workspace_bytes;
  aurora::PreparedTable table;
};

static void plan_free(delta_multi_plan* p) {
  if (!p) return;
  if (p->table.d_table) (void)hipFree(p->table.d_table);
  if (p->table.d_map) (void)hipFree(p->table.d_map);
  delete p;
}

static delta_status_t stream_device(hipStream_t stream, int* dev) {
  const hipError_t e = stream ? hipStreamGetDevice(stream, dev) : hipGetDevice(dev);
  return e == hipSuccess ? DELTA_OK : hip_fail(e, "device of the stream");
}

extern "C" {

delta_status_t delta_multi_plan_create(const uint16_t* const* prev_ptrs,
                                       const uint16_t* const* next_ptrs, const uint64_t* numels,
                                       int32_t num_tensors, hipStream_t stream,
                                       delta_multi_plan_t** out_plan) {
  if (!out_plan) return fail(DELTA_ERR_INVALID_ARG, "out_plan is NULL");
  *out_plan = nullptr;
  std::vector<SliceIn> slices;
  delta_status_t st = list_slices(prev_ptrs, next_ptrs, numels, num_tensors, slices);
  if (st != DELTA_OK) return st;
  int dev = -1;
  st = stream_device(stream, &dev);
  if (st != DELTA_OK) return st;
  delta_multi_plan* p = new (std::nothrow) delta_multi_plan();
  if (!p) return fail(DELTA_ERR_INVALID_ARG, "no host memory for the plan");
  p->device = dev;
  p->num_tensors = num_tensors;
  p->workspace_bytes = multi_workspace_bound(numels, num_tensors);
  p->table.tiles = build_descs(slices.data(), slices.size(), p->table.descs);
  p->table.d_table = nullptr;
  p->table.d_map = nullptr;
  if (p->table.tiles > 0xFFFFFFFFull / kThreads) {
    plan_free(p);
    return fail(DELTA_ERR_INVALID_ARG, "too many words for one launch");
  }
  const size_t n = p->table.descs.size();
  if (n > (size_t)kInlineDescs) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e == hipSuccess && cur != dev) e = hipSetDevice(dev);
    if (e == hipSuccess) e = hipMalloc((void**)&p->table.d_table, sizeof(TensorDesc) * n);
    if (e == hipSuccess) e = hipMalloc((void**)&p->table.d_map, 4 * p->table.tiles);
    if (cur >= 0 && cur != dev) (void)hipSetDevice(cur);
    if (e == hipSuccess)
      e = launch_upload_words((const uint64_t*)p->table.descs.data(),
                              n * sizeof(TensorDesc) / 8, (uint64_t*)p->table.d_table, stream);
    if (e == hipSuccess)
      e = launch_build_tile_map(p->table.d_table, (uint32_t)n, p->table.d_map, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) {
      plan_free(p);
      return hip_fail(e, "plan table");
    }
  }
  *out_plan = p;
  return ok();
}

delta_status_t delta_multi_plan_destroy(delta_multi_plan_t* plan) {
  if (!plan) return ok();
  hipError_t e = hipSuccess;
  if (plan->table.d_table || plan->table.d_map) {
    // calls enqueued on any stream may still read the table: finish them
    int cur = -1;
    e = hipGetDevice(&cur);
    if (e == hipSuccess && cur != plan->device) e = hipSetDevice(plan->device);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (cur >= 0 && cur != plan->device) (void)hipSetDevice(cur);
  }
  plan_free(plan);
  return e == hipSuccess ? ok() : hip_fail(e, "finishing the plan's calls");
}

size_t delta_multi_plan_workspace_bytes(const delta_multi_plan_t* plan) {
  return plan ? plan->workspace_bytes : 0;
}

delta_status_t delta_extract_multi_planned(const delta_multi_plan_t* plan, int64_t* out_idx,
                                           uint16_t* out_val, uint64_t capacity,
                                           uint64_t* d_count, uint64_t* d_tensor_offsets,
                                           void* workspace, size_t workspace_bytes,
                                           hipStream_t stream) {
  if (!plan) return fail(DELTA_ERR_INVALID_ARG, "plan is NULL");
  if (!d_count) return fail(DELTA_ERR_INVALID_ARG, "d_count is NULL");
  if (capacity > 0 && (!out_idx || !out_val))
    return fail(DELTA_ERR_INVALID_ARG, "out_idx/out_val is NULL with capacity %llu",
                (unsigned long long)capacity);
  if ((uintptr_t)out_idx % 8 || odd(out_val))
    return fail(DELTA_ERR_INVALID_ARG, "out_idx/out_val not aligned to their element size");
  int dev = -1;
  const delta_status_t st = stream_device(stream, &dev);
  if (st != DELTA_OK) return st;
  if (dev != plan->device)
    return fail(DELTA_ERR_INVALID_ARG, "the stream is on device %d, the plan on device %d", dev,
                plan->device);
  return enqueue_extract(nullptr, 0, (uint32_t)plan->num_tensors, true, out_idx, out_val,
                         capacity, d_count, d_tensor_offsets, workspace, workspace_bytes, stream,
                         nullptr, nullptr, false, &plan->table);
}

delta_status_t delta_count_changed_multi_planned(const delta_multi_plan_t* plan,
                                                 uint64_t* d_count, void* workspace,
                                                 size_t workspace_bytes, hipStream_t stream) {
  if (!plan) return fail(DELTA_ERR_INVALID_ARG, "plan is NULL");
  if (!d_count) return fail(DELTA_ERR_INVALID_ARG, "d_count is NULL");
  int dev = -1;
  const delta_status_t st = stream_device(stream, &dev);
  if (st != DELTA_OK) return st;
  if (dev != plan->device)
    return fail(DELTA_ERR_INVALID_ARG, "the stream is on device %d, the plan on device %d", dev,
                plan->device);
  return enqueue_extract(nullptr, 0, (uint32_t)plan->num_tensors, true, nullptr, nullptr, 0,
                         d_count, nullptr, workspace, workspace_bytes, stream, nullptr, nullptr,
                         true, &plan->table);
}

delta_status_t delta_extract_multi_leb128_planned(const delta_multi_plan_t* plan,
                                                  uint8_t* out_code, uint64_t code_capacity,
                                                  uint64_t* d_nbytes, uint16_t* out_val,
                                                  uint64_t capacity, uint64_t* d_count,
                                                  uint64_t* d_tensor_offsets,
                                                  uint64_t* d_tensor_byte_offsets,
                                                  void* workspace, size_t workspace_bytes,
                                                  hipStream_t stream) {
  if (!plan) return fail(DELTA_ERR_INVALID_ARG, "plan is NULL");
  if (!d_count || !d_nbytes) return fail(DELTA_ERR_INVALID_ARG, "d_count/d_nbytes is NULL");
  if (capacity > 0 && !out_val)
    return fail(DELTA_ERR_INVALID_ARG, "out_val is NULL with capacity %llu",
                (unsigned long long)capacity);
  if (odd(out_val)) return fail(DELTA_ERR_INVALID_ARG, "out_val not 2-byte aligned");
  if (code_capacity > 0 && !out_code)
    return fail(DELTA_ERR_INVALID_ARG, "out_code is NULL with code_capacity %llu",
                (unsigned long long)code_capacity);
  int dev = -1;
  const delta_status_t st = stream_device(stream, &dev);
  if (st != DELTA_OK) return st;
  if (dev != plan->device)
    return fail(DELTA_ERR_INVALID_ARG, "the stream is on device %d, the plan on device %d", dev,
                plan->device);
  const CodedOut co = {out_code, code_capacity, d_nbytes, 0, true, d_tensor_byte_offsets};
  return enqueue_extract(nullptr, 0, (uint32_t)plan->num_tensors, true, nullptr, out_val,
                         capacity, d_count, d_tensor_offsets, workspace, workspace_bytes, stream,
                         &co, nullptr, false, &plan->table);
}

delta_status_t delta_count_changed_multi(const uint16_t* const* prev_ptrs,
                                         const uint16_t* const* next_ptrs,
                                         const uint64_t* numels, int32_t num_tensors,
                                         uint64_t* d_count, void* workspace,
                                         size_t workspace_bytes, hipStream_t stream) {
  if (!d_count) return fail(DELTA_ERR_INVALID_ARG, "d_count is NULL");
  std::vector<SliceIn> slices;
  const delta_status_t st = list_slices(prev_ptrs, next_ptrs, numels, num_tensors, slices);
  if (st != DELTA_OK) return st;
  return enqueue_extract(slices.data(), slices.size(), (uint32_t)num_tensors, true, nullptr,
                         nullptr, 0, d_count, nullptr, workspace, workspace_bytes, stream,
                         nullptr, nullptr, true);
}

size_t delta_extract_multi_leb128_workspace_bytes(const uint64_t* numels, int32_t num_tensors) {
  if (num_tensors < 0 || (num_tensors > 0 && !numels)) return 0;
  return multi_workspace_bound(numels, num_tensors, true);
}

delta_status_t delta_extract_multi_leb128(const uint16_t* const* prev_ptrs,
                                          const uint16_t* const* next_ptrs,
                                          const uint64_t* numels, int32_t num_tensors,
                                          uint8_t* out_code, uint64_t code_capacity,
                                          uint64_t* d_nbytes, uint16_t* out_val,
                                          uint64_t capacity, uint64_t* d_count,
                                          uint64_t* d_tensor_offsets,
                                          uint64_t* d_tensor_byte_offsets, void* workspace,
                                          size_t workspace_bytes, hipStream_t stream) {
  if (!d_count || !d_nbytes) return fail(DELTA_ERR_INVALID_ARG, "d_count/d_nbytes is NULL");
  if (capacity > 0 && !out_val)
    return fail(DELTA_ERR_INVALID_ARG, "out_val is NULL with capacity %llu",
                (unsigned long long)capacity);
  if (odd(out_val)) return fail(DELTA_ERR_INVALID_ARG, "out_val not 2-byte aligned");
  if (code_capacity > 0 && !out_code)
    return fail(DELTA_ERR_INVALID_ARG, "out_code is NULL with code_capacity %llu",
                (unsigned long long)code_capacity);
  std::vector<SliceIn> slices;
  const delta_status_t st = list_slices(prev_ptrs, next_ptrs, numels, num_tensors, slices);
  if (st != DELTA_OK) return st;
  const CodedOut co = {out_code, code_capacity, d_nbytes, 0, true, d_tensor_byte_offsets};
  return enqueue_extract(slices.data(), slices.size(), (uint32_t)num_tensors, true, nullptr,
                         out_val, capacity, d_count, d_tensor_offsets, workspace,
                         workspace_bytes, stream, &co);
}

delta_status_t delta_extract_fused(const uint16_t* const* prev_ptrs,
                                   const uint16_t* const* next_ptrs, const uint64_t* numels,
                                   int32_t num_tensors, const int32_t* target,
                                   const uint64_t* block_offset, const uint64_t* target_numels,
                                   int32_t num_targets, int64_t* out_idx, uint16_t* out_val,
                                   uint64_t capacity, uint64_t* d_count,
                                   uint64_t* d_target_offsets, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream) {
  if (num_tensors < 0 || num_targets < 0)
    return fail(DELTA_ERR_INVALID_ARG, "negative tensor count");
  if (num_tensors > 0 && (!prev_ptrs || !next_ptrs || !numels || !target || !block_offset))
    return fail(DELTA_ERR_INVALID_ARG, "tensor arrays are NULL");
  if (num_targets > 0 && !target_numels)
    return fail(DELTA_ERR_INVALID_ARG, "target_numels is NULL");
  if (!d_count) return fail(DELTA_ERR_INVALID_ARG, "d_count is NULL");
  if (capacity > 0 && (!out_idx || !out_val))
    return fail(DELTA_ERR_INVALID_ARG, "out_idx/out_val is NULL with capacity %llu",
                (unsigned long long)capacity);
  if ((uintptr_t)out_idx % 8 || odd(out_val))
    return fail(DELTA_ERR_INVALID_ARG, "out_idx/out_val not aligned to their element size");
  // global base of every target
  std::vector<uint64_t> tbase(num_targets + 1, 0);
  for (int32_t f = 0; f < num_targets; ++f) {
    if (tbase[f] + target_numels[f] < tbase[f])
      return fail(DELTA_ERR_INVALID_ARG, "total size overflows");
    tbase[f + 1] = tbase[f] + target_numels[f];
  }
  if (tbase[num_targets] > 0 && tbase[num_targets] - 1 > 0x7FFFFFFFFFFFFFFFull)
    return fail(DELTA_ERR_INDEX_OVERFLOW, "total size exceeds int64");
  std::vector<SliceIn> slices;
  slices.reserve(num_tensors);
  for (int32_t t = 0; t < num_tensors; ++t) {
    const int32_t f = target[t];
    if (f < 0 || f >= num_targets)
      return fail(DELTA_ERR_INVALID_ARG, "tensor %d: target %d out of range", t, f);
    if (numels[t] > 0 && (!prev_ptrs[t] || !next_ptrs[t]))
      return fail(DELTA_ERR_INVALID_ARG, "tensor %d: NULL pointer", t);
    if (odd(prev_ptrs[t]) || odd(next_ptrs[t]))
      return fail(DELTA_ERR_INVALID_ARG, "tensor %d: not 2-byte aligned", t);
    if (block_offset[t] > target_numels[f] || numels[t] > target_numels[f] - block_offset[t])
      return fail(DELTA_ERR_INVALID_ARG, "tensor %d: block [%llu, +%llu) outside target %d", t,
                  (unsigned long long)block_offset[t], (unsigned long long)numels[t], f);
    slices.push_back({prev_ptrs[t], next_ptrs[t], numels[t], tbase[f] + block_offset[t],
                      (uint32_t)f, tbase[f]});
  }
  // output order is the fused index order: blocks sorted by their base
  std::stable_sort(slices.begin(), slices.end(),
                   [](const SliceIn& x, const SliceIn& y) { return x.base < y.base; });
  // the blocks must tile every target exactly (no gap, no overlap)
  uint64_t pos = 0;
  for (const SliceIn& sl : slices) {
    if (sl.base != pos)
      return fail(DELTA_ERR_INVALID_ARG, "blocks leave a gap or overlap at fused word %llu",
                  (unsigned long long)pos);
    pos += sl.n;
  }
  if (pos != tbase[num_targets])
    return fail(DELTA_ERR_INVALID_ARG, "blocks cover %llu of %llu fused words",
                (unsigned long long)pos, (unsigned long long)tbase[num_targets]);
  return enqueue_extract(slices.data(), slices.size(), (uint32_t)num_targets, true, out_idx,
                         out_val, capacity, d_count, d_target_offsets, workspace,
                         workspace_bytes, stream);
}

delta_status_t delta_apply(uint16_t* weights, uint64_t numel, delta_index_t index_type,
                           const void* idx, const uint16_t* val, uint64_t count,
                           uint32_t* d_error_flag, hipStream_t stream) {
  if (index_type != DELTA_INDEX_I32 && index_type != DELTA_INDEX_I64)
    return fail(DELTA_ERR_INVALID_ARG, "unknown index type %d", (int)index_type);
  if (count > 0 && (!idx || !val)) return fail(DELTA_ERR_INVALID_ARG, "idx/val is NULL");
  if (count > 0 && numel > 0 && !weights) return fail(DELTA_ERR_INVALID_ARG, "weights is NULL");
  if (odd(weights) || odd(val)) return fail(DELTA_ERR_INVALID_ARG, "not 2-byte aligned");
  if ((uintptr_t)idx % (index_type == DELTA_INDEX_I64 ? 8 : 4))
    return fail(DELTA_ERR_INVALID_ARG, "idx not aligned to its element size");
  hipError_t e = launch_apply(weights, numel, index_type == DELTA_INDEX_I64, idx, val, count,
                              d_error_flag, stream);
  if (e != hipSuccess) return hip_fail(e, "apply launch");
  return ok();
}

delta_status_t delta_apply_checked(uint16_t* weights, uint64_t numel, delta_index_t index_type,
                                   const void* idx, const uint16_t* val, uint64_t count,
                                   uint32_t* d_error_flag, uint64_t active_version,
                                   uint64_t base_version, hipStream_t stream) {
  if (active_version != base_version)
    return fail(DELTA_ERR_VERSION, "delta made against version %llu, active version is %llu",
                (unsigned long long)base_version, (unsigned long long)active_version);
  return delta_apply(weights, numel, index_type, idx, val, count, d_error_flag, stream);
}

// Host table of a tensor list for the apply kernels: bases[t] = first
// global index of tensor t (bases[T] = total) and the tensors' addresses.
static delta_status_t weight_table(uint16_t* const* weight_ptrs, const uint64_t* numels,
                                   int32_t num_tensors, std::vector<uint64_t>& bases,
                                   std::vector<uint64_t>& ptrs) {
  if (num_tensors < 0) return fail(DELTA_ERR_INVALID_ARG, "num_tensors < 0");
  if (num_tensors > 0 && (!weight_ptrs || !numels))
    return fail(DELTA_ERR_INVALID_ARG, "tensor arrays are NULL");
  bases.assign(num_tensors + 1, 0);
  ptrs.assign(num_tensors, 0);
  uint64_t base = 0;
  for (int32_t t = 0; t < num_tensors; ++t) {
    if (numels[t] > 0 && !weight_ptrs[t])
      return fail(DELTA_ERR_INVALID_ARG, "tensor %d: NULL pointer", t);
    if (odd(weight_ptrs[t])) return fail(DELTA_ERR_INVALID_ARG, "tensor %d: odd address", t);
    bases[t] = base;
    ptrs[t] = (uint64_t)(uintptr_t)weight_ptrs[t];
    if (base + numels[t] < base) return fail(DELTA_ERR_INVALID_ARG, "total size overflows");
    base += numels[t];
  }
  bases[num_tensors] = base;
  return DELTA_OK;
}

// Uploads the table into the start of the workspace (the layout of
// delta_apply_multi_workspace_bytes).
static hipError_t upload_weight_table(const std::vector<uint64_t>& bases,
                                      const std::vector<uint64_t>& ptrs, char* ws,
                                      uint64_t*& d_bases, uint64_t*& d_ptrs, hipStream_t stream) {
  d_bases = (uint64_t*)ws;
  d_ptrs = (uint64_t*)(ws + align_up(8 * bases.size()));
  hipError_t e = launch_upload_words(bases.data(), bases.size(), d_bases, stream);
  if (e == hipSuccess && !ptrs.empty()) e = launch_upload_words(ptrs.data(), ptrs.size(), d_ptrs, stream);
  return e;
}

delta_status_t delta_apply_multi(uint16_t* const* weight_ptrs, const uint64_t* numels,
                                 int32_t num_tensors, const int64_t* idx, const uint16_t* val,
                                 uint64_t count, uint32_t* d_error_flag, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream) {
  std::vector<uint64_t> bases, ptrs;
  delta_status_t s = weight_table(weight_ptrs, numels, num_tensors, bases, ptrs);
  if (s != DELTA_OK) return s;
  if (count > 0 && (!idx || !val)) return fail(DELTA_ERR_INVALID_ARG, "idx/val is NULL");
  if (odd(val) || ((uintptr_t)idx % 8)) return fail(DELTA_ERR_INVALID_ARG, "idx/val misaligned");
  const size_t need = delta_apply_multi_workspace_bytes(num_tensors);
  s = check_workspace(workspace, workspace_bytes, need);
  if (s != DELTA_OK) return s;
  if (count == 0) return ok();
  uint64_t *d_bases, *d_ptrs;
  hipError_t e = upload_weight_table(bases, ptrs, (char*)workspace, d_bases, d_ptrs, stream);
  if (e != hipSuccess) return hip_fail(e, "table upload launch");
  e = launch_apply_multi(d_bases, (uint16_t* const*)d_ptrs, (uint32_t)num_tensors, idx, val,
                         count, d_error_flag, stream);
  if (e != hipSuccess) return hip_fail(e, "apply_multi launch");
  return ok();
}

delta_status_t delta_apply_multi_sorted(uint16_t* const* weight_ptrs, const uint64_t* numels,
                                        int32_t num_tensors, const int64_t* idx,
                                        const uint16_t* val, uint64_t count,
                                        uint32_t* d_error_flag, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream) {
  std::vector<uint64_t> bases, ptrs;
  delta_status_t s = weight_table(weight_ptrs, numels, num_tensors, bases, ptrs);
  if (s != DELTA_OK) return s;
  if (count > 0 && (!idx || !val)) return fail(DELTA_ERR_INVALID_ARG, "idx/val is NULL");
  if (odd(val) || ((uintptr_t)idx % 8)) return fail(DELTA_ERR_INVALID_ARG, "idx/val misaligned");
  s = check_workspace(workspace, workspace_bytes,
                      delta_apply_multi_sorted_workspace_bytes(num_tensors));
  if (s != DELTA_OK) return s;
  if (count == 0) return ok();
  char* ws = (char*)workspace;
  uint64_t *d_bases, *d_ptrs;
  hipError_t e = upload_weight_table(bases, ptrs, ws, d_bases, d_ptrs, stream);
  if (e != hipSuccess) return hip_fail(e, "table upload launch");
  const uint32_t T = (uint32_t)num_tensors;
  std::vector<uint64_t> tile_first(T + 1);
  const uint64_t tiles = merge_tiles(numels, T, tile_first.data());
  if (tiles == 0 || !merge_pays(count, bases[T]) || tiles > 0xFFFFFFFFull) {
    e = launch_apply_multi(d_bases, (uint16_t* const*)d_ptrs, T, idx, val, count, d_error_flag,
                           stream);
    if (e != hipSuccess) return hip_fail(e, "apply_multi launch");
    return ok();
  }
  uint64_t* d_tile_first = (uint64_t*)(ws + delta_apply_multi_workspace_bytes(num_tensors));
  e = launch_upload_words(tile_first.data(), tile_first.size(), d_tile_first, stream);
  if (e != hipSuccess) return hip_fail(e, "tile table upload launch");
  e = launch_apply_merge(d_bases, (uint16_t* const*)d_ptrs, d_tile_first, T, tiles, idx, val,
                         count, d_error_flag, stream);
  if (e != hipSuccess) return hip_fail(e, "apply_merge launch");
  return ok();
}

// delta_apply_chain: tiles of `per_tile` entries of the largest delta, so
// that a tile of deltas of similar density stages about kChainLds indices.
struct ChainPlan {
  uint32_t ref;
  uint64_t per_tile, tiles;
  size_t deltas, pos, tile_first, total;   // workspace offsets after the weight table
};

static ChainPlan chain_plan(const uint64_t* counts, int32_t K, int32_t T) {
  ChainPlan c;
  c.ref = 0;
  for (int32_t k = 1; k < K; ++k)
    if (counts[k] > counts[c.ref]) c.ref = (uint32_t)k;
  uint64_t s = ((uint64_t)kChainLds / (uint64_t)(K + 1)) / 16 * 16;
  c.per_tile = s < 16 ? 16 : s;
  const uint64_t n_ref = K > 0 ? counts[c.ref] : 0;
  c.tiles = (n_ref + c.per_tile - 1) / c.per_tile;
  c.deltas = delta_apply_multi_workspace_bytes(T);
  c.pos = align_up(c.deltas + sizeof(ChainDelta) * (size_t)(K > 0 ? K : 1));
  c.tile_first = align_up(c.pos + 8 * (c.tiles + 1) * (uint64_t)(K > 0 ? K : 1));
  c.total = align_up(c.tile_first + 8 * ((size_t)(T > 0 ? T : 0) + 1));
  return c;
}

size_t delta_apply_chain_workspace_bytes(const uint64_t* counts, int32_t num_deltas,
                                         int32_t num_tensors) {
  if (num_deltas < 0 || num_tensors < 0 || (num_deltas > 0 && !counts)) return 0;
  return chain_plan(counts, num_deltas, num_tensors).total;
}

delta_status_t delta_apply_chain(uint16_t* const* weight_ptrs, const uint64_t* numels,
                                 int32_t num_tensors, const int64_t* const* idx_ptrs,
                                 const uint16_t* const* val_ptrs, const uint64_t* counts,
                                 int32_t num_deltas, uint32_t* d_error_flag, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream) {
  std::vector<uint64_t> bases, ptrs;
  delta_status_t s = weight_table(weight_ptrs, numels, num_tensors, bases, ptrs);
  if (s != DELTA_OK) return s;
  if (num_deltas < 0 || num_deltas > kChainMaxDeltas)
    return fail(DELTA_ERR_INVALID_ARG, "%d deltas: 0 to %d per call (compose longer chains first)",
                num_deltas, kChainMaxDeltas);
  if (num_deltas > 0 && (!idx_ptrs || !val_ptrs || !counts))
    return fail(DELTA_ERR_INVALID_ARG, "delta arrays are NULL");
  std::vector<uint64_t> table;
  uint64_t entries = 0;
  for (int32_t k = 0; k < num_deltas; ++k) {
    if (counts[k] > 0 && (!idx_ptrs[k] || !val_ptrs[k]))
      return fail(DELTA_ERR_INVALID_ARG, "delta %d: NULL pointer", k);
    if ((uintptr_t)idx_ptrs[k] % 8 || odd(val_ptrs[k]))
      return fail(DELTA_ERR_INVALID_ARG, "delta %d: idx/val misaligned", k);
    table.push_back((uint64_t)(uintptr_t)idx_ptrs[k]);
    table.push_back((uint64_t)(uintptr_t)val_ptrs[k]);
    table.push_back(counts[k]);
    entries += counts[k];
  }
  const ChainPlan c = chain_plan(counts, num_deltas, num_tensors);
  s = check_workspace(workspace, workspace_bytes, c.total);
  if (s != DELTA_OK) return s;
  if (entries == 0) return ok();
  char* ws = (char*)workspace;
  uint64_t *d_bases, *d_ptrs;
  hipError_t e = upload_weight_table(bases, ptrs, ws, d_bases, d_ptrs, stream);
  if (e != hipSuccess) return hip_fail(e, "table upload launch");
  if (num_deltas == 1) {
    e = launch_apply_multi(d_bases, (uint16_t* const*)d_ptrs, (uint32_t)num_tensors, idx_ptrs[0],
                           val_ptrs[0], counts[0], d_error_flag, stream);
    if (e != hipSuccess) return hip_fail(e, "apply_multi launch");
    return ok();
  }
  e = launch_upload_words(table.data(), table.size(), (uint64_t*)(ws + c.deltas), stream);
  if (e != hipSuccess) return hip_fail(e, "delta table upload launch");
  // a chain dense enough (all its entries together at least one word in
  // 24): the tile merge of every delta, every word read and written once
  const uint32_t T = (uint32_t)num_tensors;
  std::vector<uint64_t> tile_first(T + 1);
  const uint64_t mtiles = merge_tiles(numels, T, tile_first.data());
  if (mtiles > 0 && chain_merge_pays(entries, bases[T]) && mtiles <= 0xFFFFFFFFull) {
    uint64_t* d_tile_first = (uint64_t*)(ws + c.tile_first);
    e = launch_upload_words(tile_first.data(), tile_first.size(), d_tile_first, stream);
    if (e != hipSuccess) return hip_fail(e, "tile table upload launch");
    e = launch_apply_runs(d_bases, (uint16_t* const*)d_ptrs, d_tile_first, T, mtiles,
                          (const ChainDelta*)(ws + c.deltas), (uint32_t)num_deltas, entries,
                          bases[T], d_error_flag, stream);
    if (e != hipSuccess) return hip_fail(e, "apply_runs launch");
    return ok();
  }
  if (c.tiles > 0xFFFFFFFFull) return fail(DELTA_ERR_INVALID_ARG, "too many entries");
  ChainArgs a;
  memset(&a, 0, sizeof(a));
  a.r.deltas = (const ChainDelta*)(ws + c.deltas);
  a.r.K = (uint32_t)num_deltas;
  a.r.tiles = c.tiles;
  a.r.bsrc = idx_ptrs[c.ref];   // tiles cut at every per_tile-th index of the largest delta
  a.r.bstride = c.per_tile;
  a.r.pos = (uint64_t*)(ws + c.pos);
  a.bases = d_bases;
  a.ptrs = (uint16_t* const*)d_ptrs;
  a.T = (uint32_t)num_tensors;
  a.err = d_error_flag;
  e = launch_apply_chain(a, stream);
  if (e != hipSuccess) return hip_fail(e, "apply_chain launch");
  return ok();
}

size_t delta_leb128_encode_workspace_bytes(uint64_t count) { return enc_layout(count).total; }

size_t delta_leb128_decode_workspace_bytes(uint64_t nbytes, uint64_t capacity, uint32_t num_segs) {
  (void)capacity;
  (void)num_segs;
  return dec_layout(nbytes).total;
}

delta_status_t delta_leb128_encode(const int64_t* idx, uint64_t count,
                                   const uint64_t* d_seg_offsets, const uint64_t* d_seg_bases,
                                   uint32_t num_segs, uint8_t* out, uint64_t capacity,
                                   uint64_t* d_nbytes, uint64_t* d_seg_byte_offsets,
                                   uint32_t* d_error_flag, void* workspace, size_t workspace_bytes,
                                   hipStream_t stream) {
  if (!d_nbytes) return fail(DELTA_ERR_INVALID_ARG, "d_nbytes is NULL");
  if (count > 0 && !idx) return fail(DELTA_ERR_INVALID_ARG, "idx is NULL");
  if ((uintptr_t)idx % 8) return fail(DELTA_ERR_INVALID_ARG, "idx not 8-byte aligned");
  if (capacity > 0 && !out) return fail(DELTA_ERR_INVALID_ARG, "out is NULL with capacity > 0");
  if (num_segs > 0 && (!d_seg_offsets || !d_seg_bases))
    return fail(DELTA_ERR_INVALID_ARG, "segment arrays are NULL");
  if (d_seg_byte_offsets && num_segs == 0)
    return fail(DELTA_ERR_INVALID_ARG, "segment byte offsets need num_segs > 0");
  const EncLayout L = enc_layout(count);
  if (L.tiles > 0xFFFFFFFFull / 256) return fail(DELTA_ERR_INVALID_ARG, "too many entries");
  delta_status_t st = check_workspace(workspace, workspace_bytes, L.total);
  if (st != DELTA_OK) return st;
  char* ws = (char*)workspace;
  EncArgs a;
  memset(&a, 0, sizeof(a));
  a.idx = idx;
  a.count = count;
  a.segs = {d_seg_offsets, d_seg_bases, num_segs, 0};
  a.out = out;
  a.capacity = capacity;
  a.d_nbytes = d_nbytes;
  a.seg_byte_offsets = d_seg_byte_offsets;
  a.err = d_error_flag;
  hipError_t e = launch_leb128_encode(a, ws, L, stream);
  if (e != hipSuccess) return hip_fail(e, "leb128 encode launch");
  return ok();
}

delta_status_t delta_leb128_decode(const uint8_t* in, uint64_t nbytes,
                                   const uint64_t* d_seg_offsets, const uint64_t* d_seg_bases,
                                   uint32_t num_segs, int64_t* out_idx, uint64_t capacity,
                                   uint64_t* d_count, uint32_t* d_error_flag, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream) {
  if (!d_count) return fail(DELTA_ERR_INVALID_ARG, "d_count is NULL");
  if (nbytes > 0 && !in) return fail(DELTA_ERR_INVALID_ARG, "in is NULL");
  if (capacity > 0 && !out_idx) return fail(DELTA_ERR_INVALID_ARG, "out_idx is NULL");
  if ((uintptr_t)out_idx % 8) return fail(DELTA_ERR_INVALID_ARG, "out_idx not 8-byte aligned");
  if (num_segs > 0 && (!d_seg_offsets || !d_seg_bases))
    return fail(DELTA_ERR_INVALID_ARG, "segment arrays are NULL");
  const DecLayout L = dec_layout(nbytes);
  if (L.btiles > 0xFFFFFFFFull / 256)
    return fail(DELTA_ERR_INVALID_ARG, "stream too long");
  delta_status_t st = check_workspace(workspace, workspace_bytes, L.total);
  if (st != DELTA_OK) return st;
  char* ws = (char*)workspace;
  DecArgs a;
  memset(&a, 0, sizeof(a));
  a.in = in;
  a.nbytes = nbytes;
  a.segs = {d_seg_offsets, d_seg_bases, num_segs, 0};
  a.out = out_idx;
  a.capacity = capacity;
  a.d_count = d_count;
  a.err = d_error_flag;
  hipError_t e = launch_leb128_decode(a, L, ws, stream);
  if (e != hipSuccess) return hip_fail(e, "leb128 decode launch");
  return ok();
}

// Workspace of delta_apply_leb128_multi: the decoder's, then the tensor
// bases (T + 1) and pointers (T), then the decoded entry count.
struct ApplyLebLayout {
  size_t dec, bases, ptrs, count, total;
};
static ApplyLebLayout apply_leb_layout(uint64_t nbytes, int32_t T) {
  ApplyLebLayout L;
  L.dec = 0;
  L.bases = align_up(dec_layout(nbytes).total);
  L.ptrs = align_up(L.bases + 8 * (uint64_t)(T + 1));
  L.count = align_up(L.ptrs + 8 * (uint64_t)T);
  L.total = align_up(L.count + 8);
  return L;
}

size_t delta_apply_leb128_workspace_bytes(uint64_t nbytes, int32_t num_tensors) {
  if (num_tensors < 0) return 0;
  return apply_leb_layout(nbytes, num_tensors).total;
}

delta_status_t delta_apply_leb128_multi(uint16_t* const* weight_ptrs, const uint64_t* numels,
                                        int32_t num_tensors, const uint8_t* code, uint64_t nbytes,
                                        const uint64_t* d_seg_offsets,
                                        const uint64_t* d_seg_bases, uint32_t num_segs,
                                        const uint16_t* val, uint64_t count,
                                        uint32_t* d_error_flag, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream) {
  std::vector<uint64_t> bases, ptrs;
  delta_status_t st = weight_table(weight_ptrs, numels, num_tensors, bases, ptrs);
  if (st != DELTA_OK) return st;
  if (nbytes > 0 && !code) return fail(DELTA_ERR_INVALID_ARG, "code is NULL");
  if (count > 0 && !val) return fail(DELTA_ERR_INVALID_ARG, "val is NULL");
  if (odd(val)) return fail(DELTA_ERR_INVALID_ARG, "val not 2-byte aligned");
  const bool tensor_bases = num_segs > 0 && !d_seg_bases;
  if (num_segs > 0 && !d_seg_offsets) return fail(DELTA_ERR_INVALID_ARG, "d_seg_offsets is NULL");
  if (tensor_bases && num_segs != (uint32_t)num_tensors)
    return fail(DELTA_ERR_INVALID_ARG,
                "d_seg_bases NULL means one segment per tensor: num_segs %u, %d tensors",
                num_segs, num_tensors);
  if (nbytes == 0 && count > 0)
    return fail(DELTA_ERR_INVALID_ARG, "%llu values but an empty index stream",
                (unsigned long long)count);
  const DecLayout D = dec_layout(nbytes);
  if (D.btiles > 0xFFFFFFFFull / 256) return fail(DELTA_ERR_INVALID_ARG, "stream too long");
  const ApplyLebLayout L = apply_leb_layout(nbytes, num_tensors);
  st = check_workspace(workspace, workspace_bytes, L.total);
  if (st != DELTA_OK) return st;
  if (nbytes == 0) return ok();   // nothing to apply
  char* ws = (char*)workspace;
  hipError_t e = launch_upload_words(bases.data(), bases.size(), (uint64_t*)(ws + L.bases), stream);
  if (e == hipSuccess && num_tensors > 0)
    e = launch_upload_words(ptrs.data(), ptrs.size(), (uint64_t*)(ws + L.ptrs), stream);
  if (e != hipSuccess) return hip_fail(e, "table upload launch");
  DecArgs a;
  memset(&a, 0, sizeof(a));
  a.in = code;
  a.nbytes = nbytes;
  // with d_seg_bases NULL, segment t is based at tensor t's first global
  // index: the first T entries of the uploaded tensor bases
  a.segs = {d_seg_offsets, tensor_bases ? (const uint64_t*)(ws + L.bases) : d_seg_bases, num_segs,
            0};
  a.capacity = count;
  a.d_count = (uint64_t*)(ws + L.count);
  a.err = d_error_flag;
  a.ptrs = (uint16_t* const*)(ws + L.ptrs);
  a.tbases = (const uint64_t*)(ws + L.bases);
  a.num_tensors = (uint32_t)num_tensors;
  a.val = val;
  e = launch_leb128_decode(a, D, ws + L.dec, stream, true);
  if (e != hipSuccess) return hip_fail(e, "leb128 apply launch");
  return ok();
}

size_t delta_compose_workspace_bytes(const uint64_t* counts, int32_t num_deltas) {
  if (num_deltas < 0 || (num_deltas > 0 && !counts)) return 0;
  return chain_layout(counts, num_deltas).total;
}

delta_status_t delta_compose(const int64_t* const* idx_ptrs, const uint16_t* const* val_ptrs,
                             const uint64_t* counts, int32_t num_deltas, int64_t* out_idx,
                             uint16_t* out_val, uint64_t capacity, uint64_t* d_count,
                             uint32_t* d_error_flag, void* workspace, size_t workspace_bytes,
                             hipStream_t stream) {
  if (num_deltas < 0) return fail(DELTA_ERR_INVALID_ARG, "num_deltas < 0");
  if (num_deltas > 0 && (!idx_ptrs || !val_ptrs || !counts))
    return fail(DELTA_ERR_INVALID_ARG, "NULL host array");
  if (!d_count) return fail(DELTA_ERR_INVALID_ARG, "d_count is NULL");
  if (capacity > 0 && (!out_idx || !out_val))
    return fail(DELTA_ERR_INVALID_ARG, "NULL output with capacity > 0");
  if ((uintptr_t)out_idx % 8 || (uintptr_t)out_val % 2)
    return fail(DELTA_ERR_INVALID_ARG, "misaligned output");
  uint64_t total = 0;
  for (int32_t d = 0; d < num_deltas; ++d) {
    if (counts[d] > 0 && (!idx_ptrs[d] || !val_ptrs[d]))
      return fail(DELTA_ERR_INVALID_ARG, "delta %d: NULL pointer", d);
    if ((uintptr_t)idx_ptrs[d] % 8 || (uintptr_t)val_ptrs[d] % 2)
      return fail(DELTA_ERR_INVALID_ARG, "delta %d: misaligned", d);
    if (counts[d] > (1ull << 56) || total + counts[d] < total)
      return fail(DELTA_ERR_INVALID_ARG, "delta %d: count too large", d);
    total += counts[d];
  }
  const ChainLayout L = chain_layout(counts, num_deltas);
  delta_status_t st = check_workspace(workspace, workspace_bytes, L.total);
  if (st != DELTA_OK) return st;
  hipError_t e = launch_compose_chain(idx_ptrs, val_ptrs, counts, num_deltas, out_idx, out_val,
                                      capacity, d_count, d_error_flag, (char*)workspace, stream);
  if (e != hipSuccess) return hip_fail(e, "compose launch");
  return ok();
}

static bool layout_of(const delta_artifact_header_t* h, ArtifactLayout* L) {
  if (!h || h->seg_bytes < 32 || h->seg_bytes % 32 || h->num_tensors > (1ull << 32) ||
      h->count > (1ull << 56) || h->idx_bytes > (1ull << 60))
    return false;
  *L = artifact_layout(h->num_tensors, h->count, h->idx_bytes, h->seg_bytes);
  return true;
}

delta_status_t delta_artifact_layout(uint64_t num_tensors, uint64_t count, uint64_t idx_bytes,
                                     uint64_t seg_bytes, delta_artifact_layout_t* out) {
  if (!out) return fail(DELTA_ERR_INVALID_ARG, "out is NULL");
  delta_artifact_header_t h;
  memset(&h, 0, sizeof(h));
  h.num_tensors = num_tensors;
  h.count = count;
  h.idx_bytes = idx_bytes;
  h.seg_bytes = seg_bytes;
  ArtifactLayout L;
  if (!layout_of(&h, &L))
    return fail(DELTA_ERR_INVALID_ARG, "seg_bytes must be a multiple of 32; sizes too large");
  *out = {L.table, L.idx, L.val, L.hashes, L.total, L.num_segments};
  return ok();
}

delta_status_t delta_hash_segments(const void* data, uint64_t nbytes, uint64_t seg_bytes,
                                   uint64_t seed, uint64_t* d_hashes, hipStream_t stream) {
  if (seg_bytes < 32 || seg_bytes % 32)
    return fail(DELTA_ERR_INVALID_ARG, "seg_bytes must be a positive multiple of 32");
  if (nbytes > 0 && (!data || !d_hashes)) return fail(DELTA_ERR_INVALID_ARG, "NULL pointer");
  if ((uintptr_t)data % 8 || (uintptr_t)d_hashes % 8)
    return fail(DELTA_ERR_INVALID_ARG, "data and d_hashes must be 8-byte aligned");
  hipError_t e = launch_hash_segments((const uint8_t*)data, nbytes, seg_bytes, seed, d_hashes,
                                      stream);
  if (e != hipSuccess) return hip_fail(e, "hash launch");
  return ok();
}

delta_status_t delta_artifact_seal(void* d_artifact, size_t artifact_bytes,
                                   const delta_artifact_header_t* header, hipStream_t stream) {
  ArtifactLayout L;
  if (!layout_of(header, &L))
    return fail(DELTA_ERR_INVALID_ARG, "bad header (seg_bytes a multiple of 32, sizes)");
  if (header->index_coding > DELTA_CODING_LEB128)
    return fail(DELTA_ERR_INVALID_ARG, "unknown index coding %u", header->index_coding);
  if (!d_artifact || (uintptr_t)d_artifact % 8)
    return fail(DELTA_ERR_INVALID_ARG, "artifact must be a non-NULL, 8-byte aligned buffer");
  if (artifact_bytes < L.total)
    return fail(DELTA_ERR_CAPACITY, "artifact needs %llu bytes, buffer has %zu",
                (unsigned long long)L.total, artifact_bytes);
  delta_artifact_header_t h = *header;
  memcpy(h.magic, "AURDELTA", 8);
  h.format = DELTA_ARTIFACT_FORMAT;
  h.num_segments = L.num_segments;
  h.hash = 0;
  hipError_t e = launch_artifact_seal((uint8_t*)d_artifact, L, h, stream);
  if (e != hipSuccess) return hip_fail(e, "seal launch");
  return ok();
}

size_t delta_artifact_verify_workspace_bytes(const delta_artifact_header_t* header) {
  ArtifactLayout L;
  if (!layout_of(header, &L)) return 0;
  return align_up(8 * (L.num_segments ? L.num_segments : 1));
}

delta_status_t delta_artifact_verify(const void* d_artifact, size_t artifact_bytes,
                                     const delta_artifact_header_t* header,
                                     uint64_t* d_bad_segments, uint64_t* d_first_bad,
                                     uint32_t* d_header_bad, void* workspace,
                                     size_t workspace_bytes, hipStream_t stream) {
  ArtifactLayout L;
  if (!layout_of(header, &L)) return fail(DELTA_ERR_INVALID_ARG, "bad header");
  if (memcmp(header->magic, "AURDELTA", 8) || header->format != DELTA_ARTIFACT_FORMAT)
    return fail(DELTA_ERR_VERSION, "not an artifact of format %d", DELTA_ARTIFACT_FORMAT);
  if (header->num_segments != L.num_segments)
    return fail(DELTA_ERR_INVALID_ARG, "header says %llu segments, layout %llu",
                (unsigned long long)header->num_segments, (unsigned long long)L.num_segments);
  if (!d_artifact || (uintptr_t)d_artifact % 8 || artifact_bytes < L.total)
    return fail(DELTA_ERR_INVALID_ARG, "artifact buffer too small or misaligned");
  if (!d_bad_segments || !d_header_bad) return fail(DELTA_ERR_INVALID_ARG, "NULL result");
  delta_status_t st =
      check_workspace(workspace, workspace_bytes, delta_artifact_verify_workspace_bytes(header));
  if (st != DELTA_OK) return st;
  hipError_t e = launch_artifact_verify((const uint8_t*)d_artifact, L, header->seg_bytes,
                                        header->version, (uint64_t*)workspace, d_bad_segments,
                                        d_first_bad, d_header_bad, stream);
  if (e != hipSuccess) return hip_fail(e, "verify launch");
  return ok();
}


// ------------------------------------------------ artifact pack / activate

}  // extern "C"

namespace {

// Reads `n` bytes of device memory after the stream's work so far.
delta_status_t read_back(void* host, const void* dev, size_t n, hipStream_t stream) {
  hipError_t e = hipStreamSynchronize(stream);
  if (e == hipSuccess && n) e = hipMemcpy(host, dev, n, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "read back");
  return DELTA_OK;
}

// Workspace of delta_artifact_pack: numels [T], tensor bases [T], first
// index byte of each tensor [T + 1], the code length, the encoder's error
// flag, then the encoder's own workspace.
struct PackLayout {
  size_t numels, bases, byte_offs, nbytes, err, enc, total;
};
PackLayout pack_layout(uint64_t count, int32_t T, bool leb) {
  const uint64_t t = T > 0 ? (uint64_t)T : 0;
  PackLayout L;
  L.numels = 0;
  L.bases = align_up(L.numels + 8 * t);
  L.byte_offs = align_up(L.bases + 8 * t);
  L.nbytes = align_up(L.byte_offs + 8 * (t + 1));
  L.err = align_up(L.nbytes + 8);
  L.enc = align_up(L.err + 8);
  L.total = align_up(L.enc + (leb ? enc_layout(count).total : 0));
  return L;
}

// Workspace of delta_artifact_activate: the verify results and fresh
// segment hashes, the segment offsets [T + 1], the error flag, then the
// apply's own workspace.
struct ActivateLayout {
  size_t bad, first_bad, header_bad, err, offs, fresh, apply, total;
};
ActivateLayout activate_layout(const ArtifactLayout& A, const delta_artifact_header_t& h) {
  ActivateLayout L;
  L.bad = 0;
  L.first_bad = 8;
  L.header_bad = 16;
  L.err = 24;
  L.offs = align_up(32);
  L.fresh = align_up(L.offs + 8 * (h.num_tensors + 1));
  L.apply = align_up(L.fresh + 8 * (A.num_segments ? A.num_segments : 1));
  const size_t apply_ws = h.index_coding == DELTA_CODING_LEB128
                              ? delta_apply_leb128_workspace_bytes(h.idx_bytes, (int32_t)h.num_tensors)
                              : delta_apply_multi_workspace_bytes((int32_t)h.num_tensors);
  L.total = align_up(L.apply + apply_ws);
  return L;
}

}  // namespace

extern "C" {

size_t delta_artifact_pack_workspace_bytes(uint64_t count, int32_t num_tensors,
                                           uint32_t index_coding) {
  if (num_tensors < 0 || index_coding > DELTA_CODING_LEB128 || count > (1ull << 56)) return 0;
  return pack_layout(count, num_tensors, index_coding == DELTA_CODING_LEB128).total;
}

delta_status_t delta_artifact_pack(const int64_t* idx, const uint16_t* val, uint64_t count,
                                   const uint64_t* d_tensor_offsets, const uint64_t* numels,
                                   int32_t num_tensors, uint32_t index_coding, uint64_t version,
                                   uint64_t base_version, uint64_t seg_bytes, void* d_artifact,
                                   size_t artifact_bytes, void* workspace, size_t workspace_bytes,
                                   hipStream_t stream, delta_artifact_header_t* h_header,
                                   uint64_t* h_total_bytes) {
  if (num_tensors < 0 || (num_tensors > 0 && (!numels || !d_tensor_offsets)))
    return fail(DELTA_ERR_INVALID_ARG, "bad tensor list");
  if (count > 0 && (!idx || !val)) return fail(DELTA_ERR_INVALID_ARG, "idx/val is NULL");
  if ((uintptr_t)idx % 8 || odd(val)) return fail(DELTA_ERR_INVALID_ARG, "idx/val misaligned");
  if (index_coding > DELTA_CODING_LEB128)
    return fail(DELTA_ERR_INVALID_ARG, "unknown index coding %u", index_coding);
  if (seg_bytes < 32 || seg_bytes % 32)
    return fail(DELTA_ERR_INVALID_ARG, "seg_bytes must be a positive multiple of 32");
  if (!d_artifact || (uintptr_t)d_artifact % 8)
    return fail(DELTA_ERR_INVALID_ARG, "artifact must be a non-NULL, 8-byte aligned buffer");
  if (count > (1ull << 56)) return fail(DELTA_ERR_INVALID_ARG, "count too large");
  const bool leb = index_coding == DELTA_CODING_LEB128;
  // tensor bases (Sec. 5.1 block offsets) from the sizes
  const size_t T = (size_t)num_tensors;
  std::vector<uint64_t> nums(numels, numels + T), bases(T, 0);
  uint64_t words = 0;
  for (size_t t = 0; t < T; ++t) {
    bases[t] = words;
    if (words + nums[t] < words) return fail(DELTA_ERR_INVALID_ARG, "total size overflows");
    words += nums[t];
  }
  if (count > words) return fail(DELTA_ERR_INVALID_ARG, "more entries than words");
  const PackLayout P = pack_layout(count, num_tensors, leb);
  delta_status_t st = check_workspace(workspace, workspace_bytes, P.total);
  if (st != DELTA_OK) return st;
  char* ws = (char*)workspace;
  uint8_t* art = (uint8_t*)d_artifact;
  // the entry offsets must describe `count` entries
  if (T > 0) {
    uint64_t ends[2];
    st = read_back(&ends[0], d_tensor_offsets, 8, stream);
    if (st == DELTA_OK) st = read_back(&ends[1], d_tensor_offsets + T, 8, stream);
    if (st != DELTA_OK) return st;
    if (ends[0] != 0 || ends[1] != count)
      return fail(DELTA_ERR_INVALID_ARG, "tensor_offsets run from %llu to %llu, not 0 to %llu",
                  (unsigned long long)ends[0], (unsigned long long)ends[1],
                  (unsigned long long)count);
  } else if (count > 0) {
    return fail(DELTA_ERR_INVALID_ARG, "entries without tensors");
  }
  hipError_t e = hipSuccess;
  if (T > 0) {
    e = launch_upload_words(nums.data(), T, (uint64_t*)(ws + P.numels), stream);
    if (e == hipSuccess) e = launch_upload_words(bases.data(), T, (uint64_t*)(ws + P.bases), stream);
    if (e != hipSuccess) return hip_fail(e, "table upload launch");
  }
  // The index stream starts right after the table whatever its length; with
  // LEB128 coding its length (hence where the values go) is known only
  // after encoding.
  const ArtifactLayout L0 = artifact_layout(T, count, 0, seg_bytes);
  uint64_t idx_bytes = 8 * count;
  if (leb) {
    EncArgs a;
    memset(&a, 0, sizeof(a));
    a.idx = idx;
    a.count = count;
    // one segment per tensor, its first entry coded as its tensor-local index
    if (T > 0) a.segs = {d_tensor_offsets, (const uint64_t*)(ws + P.bases), (uint32_t)T, 0};
    a.out = art + L0.idx;
    a.capacity = artifact_bytes > L0.idx ? artifact_bytes - L0.idx : 0;
    a.d_nbytes = (uint64_t*)(ws + P.nbytes);
    a.seg_byte_offsets = T > 0 ? (uint64_t*)(ws + P.byte_offs) : nullptr;
    a.err = (uint32_t*)(ws + P.err);
    e = launch_reset((uint64_t*)(ws + P.err), nullptr, 0, stream);
    const EncLayout EL = enc_layout(count);
    if (e == hipSuccess) e = launch_leb128_encode(a, ws + P.enc, EL, stream);
    if (e != hipSuccess) return hip_fail(e, "encode launch");
    uint64_t got[2];
    st = read_back(&got[0], ws + P.nbytes, 8, stream);
    if (st == DELTA_OK) st = read_back(&got[1], ws + P.err, 8, stream);
    if (st != DELTA_OK) return st;
    if (got[1] & 0xFFFFFFFFull)
      return fail(DELTA_ERR_INVALID_ARG, "indices not strictly increasing within a tensor");
    idx_bytes = got[0];
  }
  const ArtifactLayout L = artifact_layout(T, count, idx_bytes, seg_bytes);
  if (h_total_bytes) *h_total_bytes = L.total;
  if (artifact_bytes < L.total)
    return fail(DELTA_ERR_CAPACITY, "artifact needs %llu bytes, buffer has %zu",
                (unsigned long long)L.total, artifact_bytes);
  if (!leb && count > 0)
    e = hipMemcpyAsync(art + L.idx, idx, 8 * count, hipMemcpyDeviceToDevice, stream);
  if (e == hipSuccess && count > 0)
    e = hipMemcpyAsync(art + L.val, val, 2 * count, hipMemcpyDeviceToDevice, stream);
  if (e != hipSuccess) return hip_fail(e, "stream copy");
  e = launch_artifact_table(art, L, (const uint64_t*)(ws + P.numels), d_tensor_offsets,
                            leb ? (const uint64_t*)(ws + P.byte_offs) : nullptr, (uint32_t)T,
                            idx_bytes, count, stream);
  if (e != hipSuccess) return hip_fail(e, "table launch");
  delta_artifact_header_t h;
  memset(&h, 0, sizeof(h));
  memcpy(h.magic, "AURDELTA", 8);
  h.format = DELTA_ARTIFACT_FORMAT;
  h.index_coding = index_coding;
  h.version = version;
  h.base_version = base_version;
  h.num_tensors = T;
  h.total_words = words;
  h.count = count;
  h.idx_bytes = idx_bytes;
  h.seg_bytes = seg_bytes;
  h.num_segments = L.num_segments;
  e = launch_artifact_seal(art, L, h, stream);
  if (e != hipSuccess) return hip_fail(e, "seal launch");
  st = read_back(h_header ? (void*)h_header : (void*)&h, art, sizeof(h), stream);
  if (st != DELTA_OK) return st;
  return ok();
}

size_t delta_artifact_activate_workspace_bytes(const delta_artifact_header_t* header) {
  ArtifactLayout A;
  if (!layout_of(header, &A) || header->index_coding > DELTA_CODING_LEB128) return 0;
  return activate_layout(A, *header).total;
}

delta_status_t delta_artifact_activate(const void* d_artifact, size_t artifact_bytes,
                                       const delta_artifact_header_t* header,
                                       uint16_t* const* weight_ptrs, const uint64_t* numels,
                                       int32_t num_tensors, uint64_t active_version,
                                       void* workspace, size_t workspace_bytes,
                                       hipStream_t stream) {
  ArtifactLayout A;
  if (!layout_of(header, &A) || header->index_coding > DELTA_CODING_LEB128)
    return fail(DELTA_ERR_INVALID_ARG, "bad header");
  if (memcmp(header->magic, "AURDELTA", 8) || header->format != DELTA_ARTIFACT_FORMAT)
    return fail(DELTA_ERR_VERSION, "not an artifact of format %d", DELTA_ARTIFACT_FORMAT);
  if (header->num_segments != A.num_segments)
    return fail(DELTA_ERR_INVALID_ARG, "header says %llu segments, layout %llu",
                (unsigned long long)header->num_segments, (unsigned long long)A.num_segments);
  if (!d_artifact || (uintptr_t)d_artifact % 8 || artifact_bytes < A.total)
    return fail(DELTA_ERR_INVALID_ARG, "artifact buffer too small or misaligned");
  // Sec. 5.2: a delta is activated only onto the version it was made against
  if (header->base_version != active_version)
    return fail(DELTA_ERR_VERSION, "delta of version %llu is based on %llu, active version is %llu",
                (unsigned long long)header->version, (unsigned long long)header->base_version,
                (unsigned long long)active_version);
  std::vector<uint64_t> bases, ptrs;
  delta_status_t st = weight_table(weight_ptrs, numels, num_tensors, bases, ptrs);
  if (st != DELTA_OK) return st;
  if ((uint64_t)num_tensors != header->num_tensors || bases[num_tensors] != header->total_words)
    return fail(DELTA_ERR_INVALID_ARG, "the artifact is for %llu tensors of %llu words, got %d of %llu",
                (unsigned long long)header->num_tensors, (unsigned long long)header->total_words,
                num_tensors, (unsigned long long)bases[num_tensors]);
  const ActivateLayout W = activate_layout(A, *header);
  st = check_workspace(workspace, workspace_bytes, W.total);
  if (st != DELTA_OK) return st;
  char* ws = (char*)workspace;
  const uint8_t* art = (const uint8_t*)d_artifact;
  // verify every segment hash and the artifact hash before touching the weights
  hipError_t e = launch_artifact_verify(art, A, header->seg_bytes, header->version,
                                        (uint64_t*)(ws + W.fresh), (uint64_t*)(ws + W.bad),
                                        (uint64_t*)(ws + W.first_bad),
                                        (uint32_t*)(ws + W.header_bad), stream);
  if (e != hipSuccess) return hip_fail(e, "verify launch");
  uint64_t res[3];
  st = read_back(res, ws + W.bad, 24, stream);
  if (st != DELTA_OK) return st;
  if (res[0] != 0 || (res[2] & 0xFFFFFFFFull))
    return fail(DELTA_ERR_INTEGRITY, "artifact fails its hashes: %llu segments differ (first %llu), "
                "artifact hash %s", (unsigned long long)res[0], (unsigned long long)res[1],
                (res[2] & 0xFFFFFFFFull) ? "differs" : "ok");
  // the (verified) tensor table: sizes must match, entry offsets ascending
  const size_t T = (size_t)num_tensors;
  std::vector<uint64_t> table(3 * T + 1, 0);
  st = read_back(table.data(), art + A.table, 24 * T, stream);
  if (st != DELTA_OK) return st;
  std::vector<uint64_t> offs(T + 1, 0);
  for (size_t t = 0; t < T; ++t) {
    if (table[3 * t] != numels[t])
      return fail(DELTA_ERR_INVALID_ARG, "tensor %zu: the artifact has %llu words, got %llu", t,
                  (unsigned long long)table[3 * t], (unsigned long long)numels[t]);
    offs[t] = table[3 * t + 1];
    if (offs[t] > header->count || (t > 0 && offs[t] < offs[t - 1]))
      return fail(DELTA_ERR_INVALID_ARG, "artifact table: entry offsets out of order");
  }
  offs[T] = header->count;
  if (T > 0 && offs[0] != 0) return fail(DELTA_ERR_INVALID_ARG, "artifact table: first offset");
  e = launch_reset((uint64_t*)(ws + W.err), nullptr, 0, stream);
  if (e != hipSuccess) return hip_fail(e, "reset launch");
  uint32_t* err = (uint32_t*)(ws + W.err);
  const uint16_t* val = (const uint16_t*)(art + A.val);
  if (header->index_coding == DELTA_CODING_LEB128) {
    e = launch_upload_words(offs.data(), T + 1, (uint64_t*)(ws + W.offs), stream);
    if (e != hipSuccess) return hip_fail(e, "offsets upload launch");
    // one segment per tensor, each based at its tensor's first global index
    st = delta_apply_leb128_multi(weight_ptrs, numels, num_tensors, art + A.idx, header->idx_bytes,
                                  (const uint64_t*)(ws + W.offs), nullptr, (uint32_t)T, val,
                                  header->count, err, ws + W.apply, workspace_bytes - W.apply,
                                  stream);
  } else {
    st = delta_apply_multi(weight_ptrs, numels, num_tensors, (const int64_t*)(art + A.idx), val,
                           header->count, err, ws + W.apply, workspace_bytes - W.apply, stream);
  }
  if (st != DELTA_OK) return st;
  uint64_t flag = 0;
  st = read_back(&flag, err, 8, stream);
  if (st != DELTA_OK) return st;
  if (flag & 0xFFFFFFFFull)
    return fail(DELTA_ERR_OUT_OF_RANGE, "malformed index stream or an index outside the tensors");
  return ok();
}

delta_status_t delta_chunk_segments(const uint64_t* chunk_counts, uint64_t num_chunks,
                                    uint64_t chunk_elems, uint64_t* seg_offsets,
                                    uint64_t* seg_bases) {
  if (num_chunks > 0 && (!chunk_counts || !seg_bases))
    return fail(DELTA_ERR_INVALID_ARG, "NULL host array");
  if (!seg_offsets) return fail(DELTA_ERR_INVALID_ARG, "seg_offsets is NULL");
  if (num_chunks > 0 && chunk_elems == 0) return fail(DELTA_ERR_INVALID_ARG, "chunk_elems is 0");
  if (num_chunks > 0 && num_chunks - 1 > UINT64_MAX / (chunk_elems ? chunk_elems : 1))
    return fail(DELTA_ERR_INVALID_ARG, "chunk bases overflow");
  uint64_t at = 0;
  for (uint64_t c = 0; c < num_chunks; ++c) {
    seg_offsets[c] = at;
    seg_bases[c] = c * chunk_elems;
    if (at + chunk_counts[c] < at) return fail(DELTA_ERR_INVALID_ARG, "counts overflow");
    at += chunk_counts[c];
  }
  seg_offsets[num_chunks] = at;
  return ok();
}

}  // extern "C"
