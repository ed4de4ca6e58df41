/*
 * aurora_delta.h — C ABI of an MI355X (gfx950) library for lossless sparse
 * delta checkpoints of bf16 model weights, after AuroraRL (arXiv
 * 2602.11456), Sec. 5.1 "Lossless Sparse Delta Geo-Checkpoints" and
 * Sec. 5.2 "Streaming Delta Transfer Protocol".
 *
 * The operations:
 *   extract        Compare the previous and the updated bf16 weights word
 *                  by word and keep every word whose bits changed, as two
 *                  1-D streams: the flattened positions (int32 or int64)
 *                  and the new bf16 words (Sec. 5.1 "Sparse encoding").
 *   extract_multi  The same over a list of tensors in one index space:
 *                  tensor t's positions are offset by the total size of the
 *                  tensors before it, the fixed block offsets the paper
 *                  uses to stack q/k/v or gate/up blocks (Sec. 5.1).
 *   apply          Write the streams into the flat storage of a rollout
 *                  copy in place, so that it becomes the updated weights
 *                  bit for bit (Sec. 5.1, Sec. 5.2 "activation").
 *   apply_checked  apply, refused unless the caller's active version is
 *                  the delta's declared base version (Sec. 5.2).
 *   extract_pipelined
 *                  extract_multi split into fixed-size chunks of the global
 *                  index space: one stream reads chunk after chunk, a
 *                  second finishes (and codes) each read chunk, a third
 *                  stores each finished chunk's streams into pinned host
 *                  memory (Sec. 5.2, "Overlapped extraction and transfer":
 *                  segments emitted as soon as they are encoded).
 *   leb128, compose, artifacts, fused
 *                  the gap + LEB128 index coding (Sec. 5.1), composition
 *                  of a chain of deltas (Sec. 5.4), versioned hashed
 *                  artifacts (Sec. 5.1, 5.2) and extraction straight into
 *                  fused inference tensors (Sec. 5.1).
 *
 * Conventions (all functions):
 *   - bf16 data crosses the ABI as raw uint16_t bit patterns.  "Changed"
 *     means the 16-bit patterns differ: +0 -> -0 is a change, an identical
 *     NaN word is not.  The value stream holds the NEW words (not a
 *     difference) and apply assigns them, which makes the round trip
 *     lossless and apply idempotent.
 *   - Pointers are device pointers (hipMalloc / torch CUDA tensors) unless
 *     the name starts with h_ (host memory) or the comment says "host
 *     array".  Weight pointers must be 2-byte aligned; any other alignment
 *     is accepted (16-byte loads are used where both copies allow them).
 *   - Index order is the flattened storage order of each tensor (row-major
 *     for a C-contiguous tensor).  Output indices are strictly increasing.
 *   - The caller owns all memory.  No entry point allocates device memory;
 *     scratch space is a caller-provided, 256-byte aligned `workspace`
 *     (the pipelines call it `d_staging`).
 *     The matching *_workspace_bytes function returns the recommended size.
 *     Extract also accepts a smaller workspace (down to a few tens of bytes
 *     per 8192-word tile; below that DELTA_ERR_WORKSPACE): it then keeps
 *     fewer staged entries per tile and reads the input of tiles with more
 *     changed words twice.  Results never depend on the workspace size.
 *   - Asynchrony: extract/apply functions only enqueue work on `stream`
 *     (0 = the null stream) and return.  The return status covers argument
 *     validation and launch errors.  Device-side outcomes are read after
 *     the caller synchronises:
 *       *d_count      true number of changed words, also when it exceeds
 *                     `capacity` (then only the first `capacity` entries
 *                     are written and the caller may retry larger);
 *       *d_error_flag nonzero if some index was outside [0, numel) and was
 *                     skipped.
 *   - Errors: no exception crosses the ABI; the return value is a
 *     delta_status_t and delta_last_error() holds a detail string for the
 *     calling thread.  Calls on one workspace must not overlap in time
 *     (enqueue them on one stream).
 */
#ifndef AURORA_DELTA_H
#define AURORA_DELTA_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define AURORA_DELTA_ABI_VERSION 1

typedef enum {
  DELTA_OK = 0,
  DELTA_ERR_INVALID_ARG = 1,    /* null pointer, odd address, bad count */
  DELTA_ERR_INDEX_OVERFLOW = 2, /* int32 indices asked for numel - 1 > INT32_MAX */
  DELTA_ERR_CAPACITY = 3,       /* host-synchronous calls: output did not fit */
  DELTA_ERR_OUT_OF_RANGE = 4,   /* host-synchronous calls: an index was skipped */
  DELTA_ERR_VERSION = 5,        /* apply_checked: active != base version */
  DELTA_ERR_WORKSPACE = 6,      /* workspace missing, too small or misaligned */
  DELTA_ERR_HIP = 7,            /* a HIP runtime call failed */
  DELTA_ERR_INTEGRITY = 8       /* artifact_activate: a hash does not match */
} delta_status_t;

typedef enum { DELTA_INDEX_I32 = 0, DELTA_INDEX_I64 = 1 } delta_index_t;

/* AURORA_DELTA_ABI_VERSION of the loaded library. */
int delta_abi_version(void);

/* Static text naming a status code. */
const char* delta_status_string(int status);

/* Detail text of the last failed call on this thread ("" if none). */
const char* delta_last_error(void);

/* Timing aid for benchmarks and profilers: every later extract call
 * (delta_extract, delta_extract_multi, delta_extract_fused and the
 * pipeline's chunks) records `before` and `after` on its launch stream
 * right around the launch of its scan kernel, the kernel that reads both
 * copies; hipEventElapsedTime then gives that kernel's duration.  Both
 * NULL turns it off.  Process-wide, not thread-safe: set it while no
 * extract call is being enqueued.  Returns DELTA_ERR_INVALID_ARG if only
 * one of the two is NULL. */
delta_status_t delta_set_scan_events(hipEvent_t before, hipEvent_t after);

/* Recommended workspace bytes for delta_extract over `numel` words (any
 * alignment): holds every tile's staged entries up to 12.5% changed words
 * (about numel / 2 bytes). */
size_t delta_extract_workspace_bytes(uint64_t numel);

/* Workspace bytes for delta_extract_multi over tensors of the given sizes
 * (`numels` is a host array of `num_tensors` entries). */
size_t delta_extract_multi_workspace_bytes(const uint64_t* numels, int32_t num_tensors);

/* Workspace bytes for delta_apply_multi over `num_tensors` tensors. */
size_t delta_apply_multi_workspace_bytes(int32_t num_tensors);

/*
 * delta_extract — Sec. 5.1 "Sparse encoding", one tensor.
 *   prev, next    device, `numel` words each: the bf16 bit patterns before
 *                 and after the step.
 *   index_type    DELTA_INDEX_I32 (only if numel - 1 <= INT32_MAX, else
 *                 DELTA_ERR_INDEX_OVERFLOW) or DELTA_INDEX_I64.
 *   out_idx       device, `capacity` int32 or int64 entries: positions of
 *                 the changed words, ascending.
 *   out_val       device, `capacity` words: next[out_idx[k]].
 *   d_count       device, one uint64: the true number of changed words.
 *   workspace     device scratch (delta_extract_workspace_bytes(numel)).
 * numel == 0 and prev == next are legal (count 0).  prev/next must not
 * overlap the outputs.
 */
delta_status_t delta_extract(const uint16_t* prev, const uint16_t* next, uint64_t numel,
                             delta_index_t index_type, void* out_idx, uint16_t* out_val,
                             uint64_t capacity, uint64_t* d_count, void* workspace,
                             size_t workspace_bytes, hipStream_t stream);

/* Scratch bytes of delta_extract_noalloc (one array per GPU, held by the
 * library until the process ends) and the largest numel it accepts. */
#define DELTA_NOALLOC_SCRATCH_BYTES (32u << 20)
#define DELTA_NOALLOC_MAX_WORDS (1ull << 27)

/*
 * delta_extract_noalloc — for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): delta_extract with no workspace argument.  Its scratch is a
 * fixed device array of DELTA_NOALLOC_SCRATCH_BYTES inside the library, one
 * per GPU, whose address the first call on each GPU looks up (make that
 * first call outside graph capture).  No call allocates memory.
 *   prev, next, numel, index_type, out_idx, out_val, capacity, d_count,
 *   stream        as delta_extract; outputs and results are identical.
 * numel above DELTA_NOALLOC_MAX_WORDS (2^27 words, 256 MiB per copy) is
 * refused with DELTA_ERR_WORKSPACE before anything is enqueued.  Every call
 * on one GPU shares that GPU's array, which keeps the last call's contents
 * (nothing in it needs to start at zero): calls that overlap in time on one
 * GPU (other streams, other threads) race and give wrong results; enqueue
 * them on one stream.
 */
delta_status_t delta_extract_noalloc(const uint16_t* prev, const uint16_t* next, uint64_t numel,
                                     delta_index_t index_type, void* out_idx, uint16_t* out_val,
                                     uint64_t capacity, uint64_t* d_count, hipStream_t stream);

/*
 * delta_extract_multi — Sec. 5.1, a tensor list in one index space.
 *   prev_ptrs, next_ptrs, numels
 *                 host arrays of `num_tensors` entries: device pointers of
 *                 each tensor's two copies and its number of words (0 is
 *                 allowed).  Tensor t's word i has global index
 *                 base_t + i, base_t = numels[0] + ... + numels[t-1].
 *   out_idx       device int64 [capacity]: global indices, ascending.
 *   out_val       device uint16 [capacity].
 *   d_count       device uint64: true total.
 *   d_tensor_offsets
 *                 device uint64 [num_tensors + 1] or NULL: entry t is the
 *                 output position of tensor t's first entry (= number of
 *                 entries with global index < base_t), entry T the total.
 *   workspace     delta_extract_multi_workspace_bytes(numels, num_tensors).
 */
delta_status_t delta_extract_multi(const uint16_t* const* prev_ptrs,
                                   const uint16_t* const* next_ptrs, const uint64_t* numels,
                                   int32_t num_tensors, int64_t* out_idx, uint16_t* out_val,
                                   uint64_t capacity, uint64_t* d_count,
                                   uint64_t* d_tensor_offsets, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream);

/*
 * Tensor-list plan — Sec. 5.1 block offsets, fixed once per model: the
 * per-tensor slice descriptors of delta_extract_multi (tile ranges, output
 * bases, alignment) and, for more than 16 tensors, their device table and
 * tile map, built once in device memory the plan owns.  A training loop
 * extracts the same tensors (the same pointers) every step; a planned call
 * skips the per-call table upload (about 45 us for 399 tensors).
 *
 * delta_multi_plan_create: arguments as delta_extract_multi; the tensors'
 *   pointers and sizes are copied, so the tensors must stay allocated (their
 *   contents may change) while the plan is used.  Allocates device memory
 *   on the stream's device and is host-synchronous.  *out_plan is NULL on
 *   failure.
 * delta_multi_plan_destroy: frees the plan (NULL: nothing).  With a device
 *   table it first waits for the plan's device (hipDeviceSynchronize), so
 *   calls already enqueued on any stream finish first; not during a graph
 *   capture on that device.
 * delta_multi_plan_workspace_bytes: the workspace a planned call needs
 *   (the same as delta_extract_multi_workspace_bytes); 0 for NULL.
 * delta_extract_multi_planned: delta_extract_multi over the plan's tensors
 *   (outputs, workspace and errors as there).  The stream must be on the
 *   plan's device (DELTA_ERR_INVALID_ARG otherwise).  Calls on one plan may
 *   overlap in time if each has its own workspace and outputs.
 * delta_count_changed_multi_planned, delta_extract_multi_leb128_planned:
 *   delta_count_changed_multi and delta_extract_multi_leb128 over the
 *   plan's tensors, the same way (the coded call's workspace is
 *   delta_extract_multi_leb128_workspace_bytes of the same sizes).
 */
typedef struct delta_multi_plan delta_multi_plan_t;
delta_status_t delta_multi_plan_create(const uint16_t* const* prev_ptrs,
                                       const uint16_t* const* next_ptrs, const uint64_t* numels,
                                       int32_t num_tensors, hipStream_t stream,
                                       delta_multi_plan_t** out_plan);
delta_status_t delta_multi_plan_destroy(delta_multi_plan_t* plan);
size_t delta_multi_plan_workspace_bytes(const delta_multi_plan_t* plan);
delta_status_t delta_extract_multi_planned(const delta_multi_plan_t* plan, int64_t* out_idx,
                                           uint16_t* out_val, uint64_t capacity,
                                           uint64_t* d_count, uint64_t* d_tensor_offsets,
                                           void* workspace, size_t workspace_bytes,
                                           hipStream_t stream);
delta_status_t delta_count_changed_multi_planned(const delta_multi_plan_t* plan,
                                                 uint64_t* d_count, void* workspace,
                                                 size_t workspace_bytes, hipStream_t stream);
delta_status_t delta_extract_multi_leb128_planned(const delta_multi_plan_t* plan,
                                                  uint8_t* out_code, uint64_t code_capacity,
                                                  uint64_t* d_nbytes, uint16_t* out_val,
                                                  uint64_t capacity, uint64_t* d_count,
                                                  uint64_t* d_tensor_offsets,
                                                  uint64_t* d_tensor_byte_offsets,
                                                  void* workspace, size_t workspace_bytes,
                                                  hipStream_t stream);

/*
 * delta_count_changed_multi — Sec. 5.1: the number of changed words of a
 * tensor list, i.e. the entry count of its sparse delta, without forming
 * the delta.  It runs the extract's read-and-compare and count steps only
 * (both copies read once, nothing staged or written), so a caller can size
 * the outputs exactly before extracting, and it gives the read cost alone.
 *   prev_ptrs, next_ptrs, numels, num_tensors  as for delta_extract_multi.
 *   d_count       device uint64: the total (overwritten).
 *   workspace     device, 256-byte aligned, at least
 *                 delta_extract_multi_workspace_bytes(numels, num_tensors)
 *                 bytes (the extract's workspace fits).
 * Errors: DELTA_ERR_INVALID_ARG (NULL d_count, bad tensor arguments as for
 * delta_extract_multi), DELTA_ERR_WORKSPACE, DELTA_ERR_HIP.
 */
delta_status_t delta_count_changed_multi(const uint16_t* const* prev_ptrs,
                                         const uint16_t* const* next_ptrs,
                                         const uint64_t* numels, int32_t num_tensors,
                                         uint64_t* d_count, void* workspace,
                                         size_t workspace_bytes, hipStream_t stream);

/*
 * delta_extract_fused — Sec. 5.1: the delta written under the inference
 * engine's fused names, where blocks of several training tensors are
 * stacked into one (q, k, v rows into qkv_proj; gate, up into
 * gate_up_proj) by adding a fixed block offset to each block's linear
 * indices.  The result equals delta_extract_multi over the fused tensors
 * (each the concatenation of its blocks' words) in target order, without
 * building them: indices are global over the targets (target f starts at
 * the sum of target_numels before it), d_target_offsets (nullable,
 * num_targets + 1) counts the entries before each target, so
 * delta_apply_multi on the fused weights applies it directly.
 *   prev_ptrs, next_ptrs, numels  host arrays: the training tensors.
 *   target, block_offset  host arrays per training tensor: its fused
 *                 tensor and the word offset of its block there.
 *   target_numels host array: words of every fused tensor.  The blocks
 *                 must tile every target exactly (DELTA_ERR_INVALID_ARG
 *                 otherwise).
 *   workspace     delta_extract_multi_workspace_bytes(numels, num_tensors).
 */
delta_status_t delta_extract_fused(const uint16_t* const* prev_ptrs,
                                   const uint16_t* const* next_ptrs, const uint64_t* numels,
                                   int32_t num_tensors, const int32_t* target,
                                   const uint64_t* block_offset, const uint64_t* target_numels,
                                   int32_t num_targets, int64_t* out_idx, uint16_t* out_val,
                                   uint64_t capacity, uint64_t* d_count,
                                   uint64_t* d_target_offsets, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream);

/*
 * delta_apply — Sec. 5.1 / 5.2: weights[idx[k]] = val[k] for k < count,
 * in place.  Indices must be distinct (any order); entries with an index
 * outside [0, numel) are skipped and set *d_error_flag (if not NULL) to a
 * nonzero value (the flag is only ever set, never cleared).
 *   weights       device uint16 [numel], updated in place.
 *   idx, val      device streams of `count` entries (int32 or int64 idx).
 */
delta_status_t delta_apply(uint16_t* weights, uint64_t numel, delta_index_t index_type,
                           const void* idx, const uint16_t* val, uint64_t count,
                           uint32_t* d_error_flag, hipStream_t stream);

/*
 * delta_apply_multi — the scatter over a tensor list addressed by global
 * int64 indices as produced by delta_extract_multi (same tensor order and
 * sizes).  weight_ptrs and numels are host arrays of `num_tensors`
 * entries.  workspace: delta_apply_multi_workspace_bytes(num_tensors).
 */
delta_status_t delta_apply_multi(uint16_t* const* weight_ptrs, const uint64_t* numels,
                                 int32_t num_tensors, const int64_t* idx, const uint16_t* val,
                                 uint64_t count, uint32_t* d_error_flag, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes for delta_apply_multi_sorted over `num_tensors` tensors. */
size_t delta_apply_multi_sorted_workspace_bytes(int32_t num_tensors);

/*
 * delta_apply_multi_sorted — delta_apply_multi (Sec. 5.1 scatter into the
 * flattened tensor list, Sec. 5.2 activation) for a delta whose indices are
 * strictly increasing, as delta_extract_multi writes them.  Same arguments;
 * workspace: delta_apply_multi_sorted_workspace_bytes(num_tensors).
 * When the delta holds at least one word in 32 of the tensor list, every
 * tile of 16384 words of each tensor is read once, patched in LDS with its
 * slice of the delta and written back whole (a delta that dense touches
 * nearly every 64-byte line, and a line written whole costs less than a
 * partially written one); below that density it scatters as
 * delta_apply_multi does.  Entries outside the tensor list set the flag and
 * are skipped; input out of order gives an unspecified result (no access
 * leaves the tensors) and may set the flag.
 */
delta_status_t delta_apply_multi_sorted(uint16_t* const* weight_ptrs, const uint64_t* numels,
                                        int32_t num_tensors, const int64_t* idx,
                                        const uint16_t* val, uint64_t count,
                                        uint32_t* d_error_flag, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream);

/*
 * delta_apply_checked — Sec. 5.2: a delta is activated only on top of the
 * version it was made against.  Returns DELTA_ERR_VERSION without touching
 * the weights when active_version != base_version; otherwise as
 * delta_apply.
 */
delta_status_t delta_apply_checked(uint16_t* weights, uint64_t numel, delta_index_t index_type,
                                   const void* idx, const uint16_t* val, uint64_t count,
                                   uint32_t* d_error_flag, uint64_t active_version,
                                   uint64_t base_version, hipStream_t stream);

/*
 * Gap + unsigned LEB128 index encoding — Sec. 5.1 "Sparse encoding" and the
 * figure "Delta checkpoint index encoding".  A sorted index stream keeps its
 * first entry as-is and every later entry as the difference from its
 * predecessor; each number is written as unsigned LEB128 (7 payload bits per
 * byte, least significant group first, bit 7 set on every byte but the
 * last; e.g. 198 -> C6 01).
 *
 * Segments: entries [seg_offsets[s], seg_offsets[s+1]) form segment s
 * (seg_offsets: device uint64 [num_segs + 1], nondecreasing, [0] = 0,
 * [num_segs] = count); the first entry of segment s is coded as
 * idx - seg_bases[s] (device uint64 [num_segs]).  With the tensor_offsets
 * of delta_extract_multi and the tensor bases this gives every tensor its
 * own stream of tensor-local indices, as in the paper.  num_segs = 0: one
 * segment, base 0 (the seg arrays may be NULL).
 */

/* Workspace bytes for delta_leb128_encode over `count` entries. */
size_t delta_leb128_encode_workspace_bytes(uint64_t count);

/* Workspace bytes for delta_leb128_decode of `nbytes` bytes into at most
 * `capacity` entries with `num_segs` segments (the size currently depends
 * on nbytes alone). */
size_t delta_leb128_decode_workspace_bytes(uint64_t nbytes, uint64_t capacity, uint32_t num_segs);

/*
 * delta_leb128_encode
 *   idx           device int64 [count], strictly increasing within each
 *                 segment and >= the segment's base at its first entry;
 *                 otherwise *d_error_flag is set (if not NULL) and the
 *                 offending gaps are coded as 0.
 *   out           device bytes [capacity]; *d_nbytes receives the true
 *                 length (only the first `capacity` bytes are written).
 *   d_seg_byte_offsets
 *                 device uint64 [num_segs + 1] or NULL: byte position where
 *                 each segment's numbers start, and the total.
 */
delta_status_t delta_leb128_encode(const int64_t* idx, uint64_t count,
                                   const uint64_t* d_seg_offsets, const uint64_t* d_seg_bases,
                                   uint32_t num_segs, uint8_t* out, uint64_t capacity,
                                   uint64_t* d_nbytes, uint64_t* d_seg_byte_offsets,
                                   uint32_t* d_error_flag, void* workspace, size_t workspace_bytes,
                                   hipStream_t stream);

/*
 * delta_leb128_decode — inverse of delta_leb128_encode.
 *   in            device bytes [nbytes].
 *   out_idx       device int64 [capacity]: decoded indices; *d_count gets
 *                 the number of numbers in the stream (only the first
 *                 `capacity` decoded).
 *   *d_error_flag set (if not NULL) when the stream ends inside a number or
 *                 a number does not fit 64 bits.
 */
delta_status_t delta_leb128_decode(const uint8_t* in, uint64_t nbytes,
                                   const uint64_t* d_seg_offsets, const uint64_t* d_seg_bases,
                                   uint32_t num_segs, int64_t* out_idx, uint64_t capacity,
                                   uint64_t* d_count, uint32_t* d_error_flag, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes for delta_extract_multi_leb128 over tensors of the given
 * sizes (host array). */
size_t delta_extract_multi_leb128_workspace_bytes(const uint64_t* numels, int32_t num_tensors);

/*
 * delta_extract_multi_leb128 — delta_extract_multi whose index stream leaves
 * the extract already gap + LEB128 coded (Sec. 5.1 "Sparse encoding"): the
 * int64 index stream is never formed.  One segment per tensor: the bytes
 * equal delta_leb128_encode of delta_extract_multi's indices with
 * seg_offsets = tensor_offsets and seg_bases = the tensor bases, so each
 * tensor's first entry is its tensor-local index and the rest are gaps.
 *   prev_ptrs, next_ptrs, numels, num_tensors  as delta_extract_multi.
 *   out_code      device bytes [code_capacity]: the coded indices; only the
 *                 first code_capacity bytes are written.
 *   d_nbytes      device uint64: the true code length.
 *   out_val       device words [capacity], as delta_extract_multi.
 *   d_count       device uint64: the true number of entries.
 *   d_tensor_offsets       device uint64 [num_tensors + 1] or NULL: entry
 *                 offsets, as delta_extract_multi.
 *   d_tensor_byte_offsets  device uint64 [num_tensors + 1] or NULL: byte
 *                 offset in out_code where each tensor's numbers start, and
 *                 the total (what delta_leb128_encode returns as
 *                 d_seg_byte_offsets).
 *   workspace     delta_extract_multi_leb128_workspace_bytes(numels, T).
 * Enqueues on `stream`.  At most 9 code bytes per entry (indices are below
 * 2^63); at 1% density about 1.3.
 */
delta_status_t delta_extract_multi_leb128(const uint16_t* const* prev_ptrs,
                                          const uint16_t* const* next_ptrs,
                                          const uint64_t* numels, int32_t num_tensors,
                                          uint8_t* out_code, uint64_t code_capacity,
                                          uint64_t* d_nbytes, uint16_t* out_val,
                                          uint64_t capacity, uint64_t* d_count,
                                          uint64_t* d_tensor_offsets,
                                          uint64_t* d_tensor_byte_offsets, void* workspace,
                                          size_t workspace_bytes, hipStream_t stream);

/*
 * Delta chains — Sec. 5.4, "Version-predicate join and delta catch-up": a
 * worker K versions behind replays the missed deltas D_1 .. D_K in order.
 * Apply assigns the new words, so that replay equals applying one delta
 * that holds every index of the chain with the value of the newest delta
 * that has it (the last writer wins).  delta_compose builds that delta.
 */

/* Workspace bytes for delta_apply_leb128_multi of `nbytes` code bytes onto
 * `num_tensors` tensors. */
size_t delta_apply_leb128_workspace_bytes(uint64_t nbytes, int32_t num_tensors);

/*
 * delta_apply_leb128_multi — Sec. 5.1 / 5.2 on the receiving side: apply a
 * delta whose indices arrive gap + LEB128 coded straight into the tensor
 * list, decoding them on the fly (no index stream is materialised).
 *   weight_ptrs, numels, num_tensors  as delta_apply_multi (host arrays);
 *                 the decoded indices are global over the concatenation.
 *   code, nbytes  device bytes of the coded indices.
 *   d_seg_offsets, d_seg_bases, num_segs  the segments, as for
 *                 delta_leb128_decode: one per tensor (seg_offsets =
 *                 tensor_offsets, seg_bases = tensor bases) as
 *                 delta_leb128_encode writes them for delta_extract_multi's
 *                 output, or one per chunk as the coded pipeline writes
 *                 them (delta_chunk_segments).  d_seg_bases NULL with
 *                 num_segs == num_tensors: one segment per tensor, each
 *                 based at its tensor's first global index (derived from
 *                 numels).
 *   val, count    device words [count]: entry k's new word.
 *   d_error_flag  device, nullable: set when the stream is malformed, when
 *                 it holds a number of entries other than `count`, or when
 *                 an index falls outside the tensor list (those words are
 *                 skipped).
 * Enqueues on `stream`; apply(W, delta) == delta_apply_multi(W, decode(code), val).
 */
delta_status_t delta_apply_leb128_multi(uint16_t* const* weight_ptrs, const uint64_t* numels,
                                        int32_t num_tensors, const uint8_t* code, uint64_t nbytes,
                                        const uint64_t* d_seg_offsets,
                                        const uint64_t* d_seg_bases, uint32_t num_segs,
                                        const uint16_t* val, uint64_t count,
                                        uint32_t* d_error_flag, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes for delta_compose of `num_deltas` deltas with these entry
 * counts (host array); 0 if the arguments are invalid. */
size_t delta_compose_workspace_bytes(const uint64_t* counts, int32_t num_deltas);

/*
 * delta_compose
 *   idx_ptrs, val_ptrs  host arrays of num_deltas device pointers, oldest
 *                 delta first: int64 indices (strictly increasing within
 *                 each delta, as delta_extract_multi writes them) and
 *                 16-bit words.  Unsorted input gives an unspecified result
 *                 (never an access out of bounds) and may set the flag.
 *   counts        host array: entries of each delta.
 *   out_idx, out_val  device arrays of `capacity` entries: the composed
 *                 delta, strictly increasing; *d_count gets its true size
 *                 (only the first `capacity` entries are written).
 *   d_error_flag  nullable device uint32, set on inconsistent (unsorted)
 *                 input.
 * Enqueued on `stream` without any host wait (intermediate counts stay on
 * the device).  apply(W, compose(D_1..D_K)) == apply(..apply(W, D_1).., D_K).
 */
delta_status_t delta_compose(const int64_t* const* idx_ptrs, const uint16_t* const* val_ptrs,
                             const uint64_t* counts, int32_t num_deltas, int64_t* out_idx,
                             uint16_t* out_val, uint64_t capacity, uint64_t* d_count,
                             uint32_t* d_error_flag, void* workspace, size_t workspace_bytes,
                             hipStream_t stream);

/* Workspace bytes for delta_apply_chain of `num_deltas` deltas with these
 * entry counts (host array) onto `num_tensors` tensors; 0 if the arguments
 * are invalid. */
size_t delta_apply_chain_workspace_bytes(const uint64_t* counts, int32_t num_deltas,
                                         int32_t num_tensors);

/*
 * delta_apply_chain — Sec. 5.4 catch-up in one pass: brings the tensor list
 * forward over the deltas D_1 .. D_K (oldest first) by writing every index
 * of the chain once, with the word of the newest delta that holds it.  The
 * result equals replaying the chain (delta_apply_multi of each delta in
 * order) and applying delta_compose's output, without forming the composed
 * delta.
 *   weight_ptrs, numels, num_tensors  as delta_apply_multi (host arrays).
 *   idx_ptrs, val_ptrs, counts  host arrays of num_deltas (0..16) entries:
 *                 each delta's int64 global indices (strictly increasing, as
 *                 delta_extract_multi writes them) and words, in device
 *                 memory, and its entry count.
 *   d_error_flag  device uint32 or NULL: set when an index falls outside
 *                 the tensor list (that entry is skipped) or the input is
 *                 found unsorted (the result is then unspecified, but no
 *                 access leaves the given buffers).
 *   workspace     delta_apply_chain_workspace_bytes(counts, num_deltas,
 *                 num_tensors).
 * Enqueues on `stream`.  A chain whose entries together hold at least one
 * word in 24 of the tensor list is merged tile by tile: every tile of 16384
 * words is read once, the deltas' words for it are patched in oldest first
 * and the tile is written back whole.  A sparser chain is cut into value
 * ranges holding a fixed number of entries of the largest delta, each
 * merged in LDS and its newest words scattered; deltas of very uneven
 * density stay correct but slower.
 */
delta_status_t delta_apply_chain(uint16_t* const* weight_ptrs, const uint64_t* numels,
                                 int32_t num_tensors, const int64_t* const* idx_ptrs,
                                 const uint16_t* const* val_ptrs, const uint64_t* counts,
                                 int32_t num_deltas, uint32_t* d_error_flag, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream);

/*
 * Versioned delta checkpoints — Sec. 5.1: the trainer writes each step's
 * delta as an immutable, versioned file with an integrity hash; Sec. 5.2:
 * it travels as segments that are verified against that hash, and a worker
 * activates it only onto its declared base version.
 *
 * Artifact layout (little-endian, offsets from delta_artifact_layout):
 *   header        delta_artifact_header_t (128 bytes)
 *   tensor table  num_tensors x {numel, first entry, first index byte}
 *                 (3 x uint64 each)
 *   index stream  idx_bytes: int64 global indices (DELTA_CODING_INT64) or
 *                 gap + LEB128 with one segment per tensor
 *                 (DELTA_CODING_LEB128)
 *   value stream  count x 16-bit words (8-byte aligned start)
 *   segment hashes  num_segments x uint64: XXH64 (seed = version) of each
 *                 seg_bytes piece of [tensor table, segment hashes)
 * The artifact hash is XXH64 of the segment hash table, seeded with the
 * XXH64 (seed 0) of the header's first 80 bytes.  XXH64 follows Y. Collet's
 * xxHash specification.
 */
typedef enum { DELTA_CODING_INT64 = 0, DELTA_CODING_LEB128 = 1 } delta_index_coding_t;

#define DELTA_ARTIFACT_FORMAT 1

typedef struct {
  char magic[8];          /* "AURDELTA" (written by seal) */
  uint32_t format;        /* DELTA_ARTIFACT_FORMAT (written by seal) */
  uint32_t index_coding;  /* delta_index_coding_t */
  uint64_t version;       /* the policy version this delta produces */
  uint64_t base_version;  /* the version it must be applied onto */
  uint64_t num_tensors;
  uint64_t total_words;   /* words of the whole tensor list */
  uint64_t count;         /* entries */
  uint64_t idx_bytes;     /* bytes of the index stream */
  uint64_t seg_bytes;     /* hash segment size: a multiple of 32, >= 32 */
  uint64_t num_segments;  /* written by seal */
  uint64_t hash;          /* written by seal */
  uint64_t reserved[5];
} delta_artifact_header_t;

typedef struct {
  uint64_t table, idx, val, hashes, total, num_segments;
} delta_artifact_layout_t;

/* Offsets and total size of an artifact (host only). */
delta_status_t delta_artifact_layout(uint64_t num_tensors, uint64_t count, uint64_t idx_bytes,
                                     uint64_t seg_bytes, delta_artifact_layout_t* out);

/*
 * XXH64 (seed) of each seg_bytes piece of the device buffer `data` (the last
 * piece may be shorter) into d_hashes[ceil(nbytes / seg_bytes)].  data must
 * be 8-byte aligned, seg_bytes a multiple of 32.
 */
delta_status_t delta_hash_segments(const void* data, uint64_t nbytes, uint64_t seg_bytes,
                                   uint64_t seed, uint64_t* d_hashes, hipStream_t stream);

/*
 * delta_artifact_seal — the caller has written the tensor table, the index
 * stream and the value stream into the device buffer d_artifact at the
 * layout's offsets; seal writes the header (from *header: magic, format
 * and num_segments are filled in) and the segment hash table, then the
 * artifact hash.  d_artifact 8-byte aligned, artifact_bytes >= the
 * layout's total.
 */
delta_status_t delta_artifact_seal(void* d_artifact, size_t artifact_bytes,
                                   const delta_artifact_header_t* header, hipStream_t stream);

/* Workspace bytes of delta_artifact_verify for this header. */
size_t delta_artifact_verify_workspace_bytes(const delta_artifact_header_t* header);

/*
 * delta_artifact_verify — recomputes every segment hash and the artifact
 * hash.  *header is the caller's host copy of the artifact's header (it
 * fixes the layout; a header changed on the way fails the artifact hash).
 *   d_bad_segments  device uint64: segments whose hash differs.
 *   d_first_bad     nullable device uint64: the first such segment
 *                   (UINT64_MAX if none).
 *   d_header_bad    device uint32: 1 if the artifact hash differs.
 */
delta_status_t delta_artifact_verify(const void* d_artifact, size_t artifact_bytes,
                                     const delta_artifact_header_t* header,
                                     uint64_t* d_bad_segments, uint64_t* d_first_bad,
                                     uint32_t* d_header_bad, void* workspace,
                                     size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes of delta_artifact_pack for `count` entries over
 * `num_tensors` tensors with this index coding (0 if invalid). */
size_t delta_artifact_pack_workspace_bytes(uint64_t count, int32_t num_tensors,
                                           uint32_t index_coding);

/*
 * delta_artifact_pack — Sec. 5.1: the trainer's versioned delta file, in
 * device memory, from delta_extract_multi's output: header, tensor table,
 * index stream, value stream and segment hashes, sealed (the same bytes
 * delta_artifact_seal gives for the same parts).
 *   idx, val, count   device: the global int64 indices and words of a
 *                     delta_extract_multi call, and their number.
 *   d_tensor_offsets  device uint64 [num_tensors + 1]: its tensor_offsets
 *                     (entry 0 must be 0 and entry T must be count).
 *   numels            host array [num_tensors]: the tensor list's sizes;
 *                     the tensor bases (Sec. 5.1 block offsets) and the
 *                     table are derived from them here.
 *   index_coding      DELTA_CODING_INT64 (the indices as they are) or
 *                     DELTA_CODING_LEB128 (gap + LEB128, one segment per
 *                     tensor, each tensor's first entry coded as its
 *                     tensor-local index).
 *   version, base_version, seg_bytes   the header's fields.
 *   d_artifact, artifact_bytes  device output, 8-byte aligned.
 *   workspace         delta_artifact_pack_workspace_bytes(count, T, coding).
 *   h_header          host, nullable: the sealed header (with its hash).
 *   h_total_bytes     host, nullable: the artifact's size.
 * Host-synchronous (the LEB128 stream's length decides where the values
 * go): returns when the artifact is sealed.  DELTA_ERR_CAPACITY, with
 * *h_total_bytes set, when artifact_bytes is too small; DELTA_ERR_INVALID_ARG
 * when the offsets or the order of the indices are inconsistent.
 */
delta_status_t delta_artifact_pack(const int64_t* idx, const uint16_t* val, uint64_t count,
                                   const uint64_t* d_tensor_offsets, const uint64_t* numels,
                                   int32_t num_tensors, uint32_t index_coding, uint64_t version,
                                   uint64_t base_version, uint64_t seg_bytes, void* d_artifact,
                                   size_t artifact_bytes, void* workspace, size_t workspace_bytes,
                                   hipStream_t stream, delta_artifact_header_t* h_header,
                                   uint64_t* h_total_bytes);

/* Workspace bytes of delta_artifact_activate for this header (0 if the
 * header is invalid). */
size_t delta_artifact_activate_workspace_bytes(const delta_artifact_header_t* header);

/*
 * delta_artifact_activate — Sec. 5.2 staged activation: a worker applies a
 * received artifact only if it is intact and was made against the version
 * the worker holds.
 *   d_artifact, artifact_bytes, header  the artifact in device memory and
 *                     the caller's host copy of its header (which fixes
 *                     the layout; a changed header fails the artifact hash).
 *   weight_ptrs, numels, num_tensors  the rollout copy (host arrays), in
 *                     the artifact's tensor order; updated in place.
 *   active_version    the version the weights hold now.
 * Checks, in this order, before any weight is written: the header's base
 * version against active_version (DELTA_ERR_VERSION, nothing enqueued);
 * the tensor count and sizes (DELTA_ERR_INVALID_ARG); every segment hash
 * and the artifact hash (DELTA_ERR_INTEGRITY).  Then the delta is applied
 * (LEB128 indices decoded inside the apply).  Host-synchronous; a malformed
 * index stream or an index outside the tensors gives
 * DELTA_ERR_OUT_OF_RANGE after the other words were written.
 */
delta_status_t delta_artifact_activate(const void* d_artifact, size_t artifact_bytes,
                                       const delta_artifact_header_t* header,
                                       uint16_t* const* weight_ptrs, const uint64_t* numels,
                                       int32_t num_tensors, uint64_t active_version,
                                       void* workspace, size_t workspace_bytes,
                                       hipStream_t stream);

/* Options of the chunked pipeline. */
typedef struct {
  uint64_t chunk_elems; /* words of the global index space per chunk (> 0) */
  int32_t num_streams;  /* staging slots and streams, 1..16 */
  int32_t reserved;
} delta_pipeline_opts_t;

/* Device staging bytes delta_extract_pipelined needs: per stream, one
 * chunk's worst-case output plus its workspace, and the running totals and
 * per-chunk counts. */
size_t delta_pipeline_staging_bytes(const uint64_t* numels, int32_t num_tensors,
                                    const delta_pipeline_opts_t* opts);

/*
 * delta_extract_pipelined — Sec. 5.2: extract_multi over the tensor list,
 * chunk by chunk, with each chunk's (idx, val) stored into pinned host
 * memory as soon as that chunk is done, while later chunks are extracted.
 * The host output equals delta_extract_multi's.
 *   streams       host array of S = opts->num_streams HIP streams, and S
 *                 staging slots.  streams[0] runs the pass over the weights
 *                 of every chunk, one after the other; streams[1] the
 *                 kernels that finish a chunk once it has been read;
 *                 streams[2] delivers the chunks in order, one kernel per
 *                 chunk (with S >= 4, per two chunks) storing into the
 *                 host arrays.  S == 2: streams[0]
 *                 also finishes the chunks, streams[1] delivers; S == 1:
 *                 everything in order on streams[0].  Streams past the
 *                 third are not used (more streams than hardware queues
 *                 serialise).
 *   d_staging     device scratch of delta_pipeline_staging_bytes(...): a
 *                 ring of S chunk slots plus the running totals.
 *   h_idx, h_val  pinned host arrays (hipHostMalloc / pin_memory) of
 *                 h_capacity entries; kernels store into them, so pageable
 *                 memory is refused with DELTA_ERR_INVALID_ARG.
 *   h_count       host: the true total.
 * The streams start on the chunks at once and wait for no other stream:
 * writes to the weights or the staging queued elsewhere must have finished
 * (the Python binding synchronises its current stream first).
 * Host-synchronous: returns after every store has landed.  Returns
 * DELTA_ERR_CAPACITY (with *h_count = true total, the first h_capacity
 * entries written) if the output did not fit.
 */
delta_status_t delta_extract_pipelined(const uint16_t* const* prev_ptrs,
                                       const uint16_t* const* next_ptrs, const uint64_t* numels,
                                       int32_t num_tensors, const delta_pipeline_opts_t* opts,
                                       hipStream_t* streams, void* d_staging,
                                       size_t staging_bytes, int64_t* h_idx, uint16_t* h_val,
                                       uint64_t h_capacity, uint64_t* h_count);

/* Device staging bytes delta_extract_pipelined_leb128 needs: per stream,
 * one chunk's worst-case values and code bytes plus its workspace (no
 * index stream: the extract writes the code itself), and the running
 * totals and per-chunk counts. */
size_t delta_pipeline_leb128_staging_bytes(const uint64_t* numels, int32_t num_tensors,
                                           const delta_pipeline_opts_t* opts);

/*
 * delta_extract_pipelined_leb128 — the Sec. 5.2 pipeline with the index
 * stream gap + LEB128 coded on the GPU before it crosses the host link
 * (Sec. 5.1 encoding; at 1% density about 1.3 bytes per index instead of
 * 8).  Each chunk is one segment of the coded stream, based at the chunk's
 * first word (c * chunk, chunk = min(opts->chunk_elems, total words)):
 * delta_leb128_decode with seg_offsets = prefix sums of h_chunk_counts and
 * seg_bases[c] = c * chunk returns delta_extract_multi's indices exactly.
 *   streams, d_staging  as delta_extract_pipelined (the kernels that
 *                 finish a chunk write its code into its slot).
 *   h_bytes       pinned host bytes [h_bytes_capacity]: the coded indices.
 *   h_val         pinned host words [h_val_capacity]: as delta_extract_multi.
 *   h_chunk_counts host array (any memory) [h_num_chunks >=
 *                 ceil(total / chunk)]: entries of each chunk.
 *   h_count, h_nbytes  host: entry and byte totals.
 * Host-synchronous.  DELTA_ERR_CAPACITY (totals set, what fits written)
 * when either output does not fit.
 */
delta_status_t delta_extract_pipelined_leb128(
    const uint16_t* const* prev_ptrs, const uint16_t* const* next_ptrs, const uint64_t* numels,
    int32_t num_tensors, const delta_pipeline_opts_t* opts, hipStream_t* streams,
    void* d_staging, size_t staging_bytes, uint8_t* h_bytes, uint64_t h_bytes_capacity,
    uint16_t* h_val, uint64_t h_val_capacity, uint64_t* h_chunk_counts, uint64_t h_num_chunks,
    uint64_t* h_count, uint64_t* h_nbytes);

/*
 * delta_chunk_segments — the segments of a coded pipeline's index stream
 * for delta_leb128_decode and delta_apply_leb128_multi (Sec. 5.2: each
 * chunk is a segment of its own): chunk c starts at entry seg_offsets[c]
 * (the counts of the chunks before it; seg_offsets[num_chunks] = total)
 * and is based at word c * chunk_elems.  Host arrays: chunk_counts
 * [num_chunks], seg_offsets [num_chunks + 1], seg_bases [num_chunks].
 */
delta_status_t delta_chunk_segments(const uint64_t* chunk_counts, uint64_t num_chunks,
                                    uint64_t chunk_elems, uint64_t* seg_offsets,
                                    uint64_t* seg_bases);

#ifdef __cplusplus
}
#endif

#endif /* AURORA_DELTA_H */
