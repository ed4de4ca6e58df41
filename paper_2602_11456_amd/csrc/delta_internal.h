// Internal definitions shared by the library's host code and kernels.
// Not part of the public ABI (that is include/aurora_delta.h).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <vector>

#include <hip/hip_runtime.h>

#include "aurora_delta.h"

namespace aurora {

// ---------------------------------------------------------------------------
// Extract tiling.
//
// A "group" is 8 consecutive bf16 words that sit in one aligned 16-byte line
// segment, so each lane reads a group of each copy with one 16-byte load.
// A workgroup has 4 wavefronts of 64 lanes; each wavefront handles
// kChunks consecutive runs of 64 groups (one run per unrolled load), so a
// tile is 4 * kChunks * 64 groups = 8192 words with kChunks = 4.
// Tiles never span tensors.
// ---------------------------------------------------------------------------
constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kChunks = 4;
constexpr int kGroupsPerWave = kChunks * 64;
constexpr int kGroupsPerTile = kWaves * kGroupsPerWave;
constexpr int kElemsPerTile = kGroupsPerTile * 8;
// Tiles per scan group (one wavefront sums / scans a group's counts).
constexpr int kTilesPerGroup = 64;
// Staging slot of a tile, in 4-byte entries.  The default holds a tile
// with 12.5% of its words changed; a smaller workspace gives smaller slots
// (down to the minimum), and a tile that overflows its slot is read again
// when the output is written.
constexpr uint32_t kDefaultStageCap = 1024;
constexpr uint32_t kMinStageCap = 16;
// Entries between the end of a slot's capacity and the next slot.  None:
// padding the 4 KiB slot stride by 64 bytes (to spread slot starts over
// the HBM channels) measured slower, and packing the slots densely no
// faster.
constexpr uint32_t kSlotPad = 0;
// The stage kernel gathers a tile's entries in LDS before writing its slot;
// the area holds a whole tile.  Its size (32 KiB) also caps residency at
// four stage workgroups per CU: with eight, the extra loads in flight only
// add contention in the memory system (measured 3% slower).
constexpr int kLdsStage = kElemsPerTile;

// One tensor (or a slice of one) as the extract kernels see it.
struct TensorDesc {
  const uint16_t* prev;   // first word of the slice
  const uint16_t* next;
  uint64_t n;             // words in the slice
  uint64_t base;          // output index of word 0 of the slice
  uint64_t first_tile;    // first tile id of the slice
  uint32_t head;          // words between the 16-byte boundary below prev and prev
  uint32_t vec;           // 1: prev and next share alignment, 16-byte loads
  uint32_t off_lo;        // first tensor_offsets slot written by this slice's first tile
  uint32_t slot;          // the caller's tensor index of this slice
  uint64_t seg_base;      // output index of word 0 of the tensor holding the slice
};
static_assert(sizeof(TensorDesc) == 64, "TensorDesc layout");

constexpr size_t kAlign = 256;
__host__ __device__ constexpr size_t align_up(size_t x, size_t a = kAlign) { return (x + a - 1) / a * a; }

// Words between the 16-byte boundary at or below p and p (p is 2-aligned).
__host__ __device__ inline uint32_t head_words(const void* p) {
  return (uint32_t)(((uintptr_t)p & 15u) >> 1);
}

__host__ __device__ inline uint64_t tiles_for(uint64_t n, uint32_t head) {
  if (n == 0) return 0;
  uint64_t groups = (n + head + 7) / 8;
  return (groups + kGroupsPerTile - 1) / kGroupsPerTile;
}

// Upper bound on tiles for n words at any alignment.
__host__ __device__ inline uint64_t tiles_bound(uint64_t n) { return tiles_for(n, 7); }

__host__ __device__ inline uint64_t groups_for(uint64_t tiles) {
  return (tiles + kTilesPerGroup - 1) / kTilesPerGroup;
}

// Workspace layout of one extract call over `tiles` tiles of `tensors`
// slices (all offsets 256-byte aligned):
//   counts      uint32 [tiles]       kept words per tile
//   group_sum   uint64 [groups]
//   group_excl  uint64 [groups]      output offset of each group
//   map         uint32 [tiles]       tile -> slice row (tensor lists)
//   table       TensorDesc [tensors]
//   coded output only (see CodedOut):
//   tile_rec    uint64 [tiles]       kept words, code bytes of the gaps between them,
//                                    offsets of the first and last (coded stage record)
//   group_bexcl uint64 [groups]      code bytes before each group
//   group_prev  int64 [groups]       index the group's first entry is coded against
//   group_first_local int64 [groups] tensor-local index of the group's first entry
//   stage       uint32 [tiles * cap] per-tile staging slots
struct WorkspaceLayout {
  size_t counts, group_sum, group_excl, map, table, tile_rec, group_bexcl, group_prev,
      group_first_local, stage, fixed;
};

inline WorkspaceLayout workspace_layout(uint64_t tiles, uint64_t tensors, bool coded = false) {
  WorkspaceLayout w;
  const uint64_t groups = groups_for(tiles);
  w.counts = 0;
  w.group_sum = align_up(w.counts + 4 * tiles);
  w.group_excl = align_up(w.group_sum + 8 * groups);
  w.map = align_up(w.group_excl + 8 * groups);
  w.table = align_up(w.map + 4 * tiles);
  w.tile_rec = align_up(w.table + sizeof(TensorDesc) * tensors);
  w.group_bexcl = align_up(w.tile_rec + (coded ? 8 * tiles : 0));
  w.group_prev = align_up(w.group_bexcl + (coded ? 8 * groups : 0));
  w.group_first_local = align_up(w.group_prev + (coded ? 8 * groups : 0));
  w.stage = align_up(w.group_first_local + (coded ? 8 * groups : 0));
  w.fixed = w.stage;
  return w;
}

// Bytes for a given slot capacity.
inline size_t workspace_bytes(uint64_t tiles, uint64_t tensors, uint32_t cap, bool coded = false) {
  return align_up(workspace_layout(tiles, tensors, coded).fixed +
                  4ull * (cap + kSlotPad) * tiles);
}

// Slot capacity a workspace of `have` bytes affords (0 if below the minimum).
inline uint32_t stage_cap_for(size_t have, uint64_t tiles, uint64_t tensors, bool coded = false) {
  const WorkspaceLayout w = workspace_layout(tiles, tensors, coded);
  if (tiles == 0) return kMinStageCap;
  if (have < w.fixed) return 0;
  uint64_t stride = (have - w.fixed) / (4 * tiles);
  if (stride < kSlotPad + kMinStageCap) return 0;
  uint64_t cap = stride - kSlotPad;
  return cap > (uint64_t)kElemsPerTile ? (uint32_t)kElemsPerTile : (uint32_t)cap;
}

// Small host tables (tensor descriptors, bases, pointers) reach device
// memory as kernel arguments, in batches of 64-bit words, so no host buffer
// has to outlive the call and nothing is copied through a DMA engine.
constexpr int kWordBatch = 320;
struct WordBatch {
  uint64_t count;
  uint64_t w[kWordBatch];
};

// ---------------------------------------------------------------------------
// Launchers (defined in extract.hip / apply.hip).  They enqueue on `stream`
// and return the HIP error of the launch.
// ---------------------------------------------------------------------------
// Slices passed inside the kernel arguments when there are at most this
// many (no table upload, no tile map).
constexpr int kInlineDescs = 16;

struct ExtractArgs {
  const TensorDesc* table;     // device table, or nullptr: the slices are in `inl`
  const uint32_t* tile_map;    // device (with table) or nullptr
  TensorDesc inl[kInlineDescs];   // used when table == nullptr
  uint32_t num_inline;
  uint64_t num_tiles;
  uint32_t num_tensors;
  uint32_t stage_cap;          // entries a staging slot holds
  uint32_t stage_stride;       // entries between slot starts (stage_cap + kSlotPad)
  void* out_idx;
  uint16_t* out_val;
  uint64_t capacity;
  uint64_t* d_count;
  uint64_t* d_tensor_offsets;  // nullable
  uint32_t* counts;
  uint64_t* group_sum;
  uint64_t* group_excl;
  uint32_t* stage;
  // Coded output (launch_extract_coded): no indices; the kept positions
  // leave gap + LEB128 coded, as one segment whose first entry is coded
  // against code_base, or (seg_per_tensor) as one segment per tensor whose
  // first entry is coded as its tensor-local index.  Per-tile and per-group
  // tables as in WorkspaceLayout.
  uint64_t* tile_rec;
  uint64_t* group_bexcl;
  int64_t* group_prev;
  uint8_t* code_out;
  uint64_t code_capacity;
  uint64_t* d_nbytes;
  int64_t code_base;
  uint32_t seg_per_tensor;
  int64_t* group_first_local;
  uint64_t* d_tensor_byte_offsets;   // nullable (seg_per_tensor): first code byte of each tensor
};

hipError_t launch_reset(uint64_t* d_count, uint64_t* d_offsets, uint32_t num_offsets,
                        hipStream_t stream);
hipError_t launch_upload_words(const uint64_t* host_words, size_t nwords, uint64_t* dst,
                               hipStream_t stream);
hipError_t launch_build_tile_map(const TensorDesc* table, uint32_t num_tensors,
                                 uint32_t* tile_map, hipStream_t stream);
// Exclusive scan of per-tile counts in groups of kTilesPerGroup tiles:
// group_sum / group_excl get one entry per group, *d_total the sum.
hipError_t launch_group_scan(const uint32_t* counts, uint64_t num_tiles, uint64_t* group_sum,
                             uint64_t* group_excl, uint64_t* d_total, hipStream_t stream);
hipError_t launch_group_scan(const uint64_t* counts, uint64_t num_tiles, uint64_t* group_sum,
                             uint64_t* group_excl, uint64_t* d_total, hipStream_t stream);
// Where the kernels after the stage kernel (the pass that reads both
// copies) run: `staged` is recorded on the launch stream right after it and
// `rest` waits for it and takes the scan and finalize kernels.
struct StageSplit {
  hipEvent_t staged;
  hipStream_t rest;
};

// all_vec: every slice has prev and next at the same 16-byte alignment.
// split: nullable, as above.
hipError_t launch_extract(const ExtractArgs& a, bool idx64, bool all_vec, hipStream_t stream,
                          const StageSplit* split = nullptr);

// A single-tensor call over at most this many tiles finalizes each tile in
// its own workgroup (two launches in all, no group scan).
constexpr uint64_t kSmallTiles = 1024;

// Count only: the scan and the tile counts, then the group sums and scan
// that leave the total in *a.d_count; nothing is staged or written.
hipError_t launch_count(const ExtractArgs& a, bool all_vec, hipStream_t stream);

// The same extract with coded output: values to out_val, the gap + LEB128
// code of the positions to code_out, *d_count and *d_nbytes.
hipError_t launch_extract_coded(const ExtractArgs& a, bool all_vec, hipStream_t stream,
                                const StageSplit* split = nullptr);

hipError_t launch_apply(uint16_t* w, uint64_t n, bool idx64, const void* idx,
                        const uint16_t* val, uint64_t count, uint32_t* err,
                        hipStream_t stream);
hipError_t launch_apply_multi(const uint64_t* bases, uint16_t* const* ptrs, uint32_t T,
                              const int64_t* idx, const uint16_t* val, uint64_t count,
                              uint32_t* err, hipStream_t stream);
// The tile-merge apply of a sorted delta (apply.hip): merge_tiles gives the
// number of tiles over the tensors and, when tile_first is not NULL, each
// tensor's first tile (T + 1 entries); merge_pays says whether a delta of
// `count` entries over `words` words is dense enough for it.
uint64_t merge_tiles(const uint64_t* numels, uint32_t T, uint64_t* tile_first);
bool merge_pays(uint64_t count, uint64_t words);
hipError_t launch_apply_merge(const uint64_t* bases, uint16_t* const* ptrs,
                              const uint64_t* tile_first, uint32_t T, uint64_t tiles,
                              const int64_t* idx, const uint16_t* val, uint64_t count,
                              uint32_t* err, hipStream_t stream);

// Catch-up in one pass (delta_apply_chain): the chain's deltas, oldest
// first, in a device table; tiles of `per_tile` entries of the reference
// (largest) delta; pos = (tiles + 1) x K split positions (workspace).
constexpr int kChainMaxDeltas = 16;
constexpr uint32_t kChainLds = 2048;   // indices a tile stages in LDS
struct ChainDelta {
  const int64_t* idx;
  const uint16_t* val;
  uint64_t n;
};
static_assert(sizeof(ChainDelta) == 24, "uploaded as three 64-bit words per delta");
// The tiles of a chain (chain.h): boundary b (0 < b < tiles) is
// bsrc[b * bstride].
struct ChainRuns {
  const ChainDelta* deltas;   // device [K]
  uint32_t K;
  uint64_t tiles;
  const int64_t* bsrc;
  uint64_t bstride;
  uint64_t* pos;              // [(tiles + 1) * K]: entries of delta k before tile t
};
struct ChainArgs {
  ChainRuns r;
  const uint64_t* bases;      // device [T + 1]
  uint16_t* const* ptrs;      // device [T]
  uint32_t T;
  uint32_t* err;
};
hipError_t launch_apply_chain(const ChainArgs& a, hipStream_t stream);
// The tile merge of a chain of K (<= kChainMaxDeltas) sorted deltas
// (apply.hip): `entries` in all over `words` words; tiles and tile_first as
// for launch_apply_merge.  chain_merge_pays says whether a chain is dense
// enough for it (from one entry per 24 words; the single-delta merge pays
// from one in 32, as the chain's other path costs more per entry than the
// plain scatter but its merge more per tile).
hipError_t launch_apply_runs(const uint64_t* bases, uint16_t* const* ptrs,
                             const uint64_t* tile_first, uint32_t T, uint64_t tiles,
                             const ChainDelta* deltas, uint32_t K, uint64_t entries,
                             uint64_t words, uint32_t* err, hipStream_t stream);
bool chain_merge_pays(uint64_t entries, uint64_t words);
hipError_t launch_chain_split(const ChainRuns& r, hipStream_t stream);

// One slice of a tensor list for enqueue_extract: `n` words of both copies
// whose word 0 has output index `base`; `tensor` is the caller's index and
// `seg_base` the output index of that tensor's word 0.
struct SliceIn {
  const uint16_t* prev;
  const uint16_t* next;
  uint64_t n;
  uint64_t base;
  uint32_t tensor;
  uint64_t seg_base;
};

// Coded output of enqueue_extract: the positions gap + LEB128 coded, at
// most `capacity` bytes at `out`, the length in *d_nbytes; no index stream.
// One segment whose first entry is coded relative to `base`, or
// (per_tensor) one segment per tensor, each tensor's first entry coded as
// its tensor-local index; then d_offsets (entries) and d_byte_offsets
// (bytes, nullable) get num_tensors + 1 entries.
struct CodedOut {
  uint8_t* out;
  uint64_t capacity;
  uint64_t* d_nbytes;
  int64_t base;
  bool per_tensor;
  uint64_t* d_byte_offsets;
};

// The slice descriptors of a tensor list and, past kInlineDescs of them,
// their device table and tile map, built once for many calls (a
// delta_multi_plan).
struct PreparedTable {
  std::vector<TensorDesc> descs;   // host copy
  uint64_t tiles;
  TensorDesc* d_table;             // nullptr when the descriptors go inline
  uint32_t* d_map;
};

// Builds the slice table in `workspace`, then enqueues the extract kernels
// on `stream` (abi.hip).  Empty slices are skipped; d_offsets (nullable)
// has num_tensors + 1 entries.  With `coded`, out_idx, idx64 and d_offsets
// are unused and the workspace follows the coded layout.  `split` as for
// launch_extract (with nothing to read, split->rest still waits for the
// launch stream).  With `count_only`, only *d_count is written (outputs,
// d_offsets, coded and split unused).  With `prepared` the slices come
// from it (slices and num_slices unused) and nothing is uploaded.  Sets
// the error text on failure.
delta_status_t enqueue_extract(const SliceIn* slices, size_t num_slices, uint32_t num_tensors,
                               bool idx64, void* out_idx, uint16_t* out_val, uint64_t capacity,
                               uint64_t* d_count, uint64_t* d_offsets, void* workspace,
                               size_t workspace_bytes, hipStream_t stream,
                               const CodedOut* coded = nullptr,
                               const StageSplit* split = nullptr, bool count_only = false,
                               const PreparedTable* prepared = nullptr);

// Delta chain composition (compose.hip): workspace layout for `K` deltas
// of the given counts, and the enqueue of the whole chain on `stream`.
struct ChainLayout {
  size_t scratch, counts, inter, total;
  uint64_t rounds;
};
ChainLayout chain_layout(const uint64_t* counts, int32_t K);
hipError_t launch_compose_chain(const int64_t* const* idx, const uint16_t* const* val,
                                const uint64_t* counts, int32_t K, int64_t* out_idx,
                                uint16_t* out_val, uint64_t capacity, uint64_t* d_count,
                                uint32_t* err, char* ws, hipStream_t stream);

// The timing aid of delta_set_scan_events: records the "before" (0) or
// "after" (1) event on `stream` if it is set (abi.hip).
hipError_t record_scan_event(int which, hipStream_t stream);

// Thread-local detail text behind delta_last_error() (abi.hip).
void set_error(const char* fmt, ...) __attribute__((format(printf, 1, 2)));
void clear_error();

}  // namespace aurora
