// Internal definitions shared by the library's host code and kernels.
// Not part of the public ABI (that is include/aurora_delta.h).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime.h>

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
// Kept entries a tile stages in LDS before writing them out (4 bytes each);
// tiles with more changed words re-read their data to write.
constexpr int kStageCap = 4096;

// Tile state word of the decoupled look-back: the top two bits say what the
// low 62 bits hold.  One 64-bit word is written and read with single
// atomic accesses, so a reader never sees a flag without its value.
constexpr uint64_t kStateEmpty = 0;
constexpr uint64_t kStateAggregate = 1ull << 62;   // count of this tile only
constexpr uint64_t kStatePrefix = 2ull << 62;      // count of tiles 0..this
constexpr uint64_t kStateFlagMask = 3ull << 62;
constexpr uint64_t kStateValueMask = (1ull << 62) - 1;

// One tensor (or a slice of one) as the extract kernel sees it.
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
  uint64_t pad1;
};
static_assert(sizeof(TensorDesc) == 64, "TensorDesc layout");

// Device-side control words at the start of every workspace.
struct Control {
  uint32_t fallbacks;     // look-back waits that ended in counting a tile directly
  uint32_t pad[63];
};
static_assert(sizeof(Control) == 256, "Control layout");

constexpr size_t kAlign = 256;
__host__ __device__ inline size_t align_up(size_t x, size_t a = kAlign) { return (x + a - 1) / a * a; }

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

// Workspace layout (multi-tensor form; the single-tensor form uses the same
// layout with one table entry):
//   [0, 256)                     Control
//   [256, +8*tiles)              tile states
//   [.., +4*tiles)               tile -> tensor map
//   [.., +64*T)                  TensorDesc table
struct WorkspaceLayout {
  size_t states, map, table, total;
};

inline WorkspaceLayout workspace_layout(uint64_t tiles, uint64_t tensors) {
  WorkspaceLayout w;
  w.states = sizeof(Control);
  w.map = align_up(w.states + 8 * tiles);
  w.table = align_up(w.map + 4 * tiles);
  w.total = align_up(w.table + sizeof(TensorDesc) * tensors);
  return w;
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
struct ExtractArgs {
  const TensorDesc* table;     // device (multi) or nullptr (single)
  const uint32_t* tile_map;    // device (multi) or nullptr (single)
  TensorDesc single;           // used when table == nullptr
  uint64_t num_tiles;
  uint32_t num_tensors;
  void* out_idx;
  uint16_t* out_val;
  uint64_t capacity;
  uint64_t* d_count;
  uint64_t* d_tensor_offsets;  // nullable
  uint64_t* states;
  Control* ctrl;
  uint32_t spin_limit;         // look-back polls before counting a silent predecessor
};

// Default look-back patience; AURORA_DELTA_SPIN_LIMIT overrides it (tests
// set 0 to drive every wait through the fallback).
constexpr uint32_t kDefaultSpinLimit = 128;
uint32_t spin_limit_from_env();

hipError_t launch_reset(Control* ctrl, uint64_t* states, uint64_t num_tiles,
                        uint64_t* d_count, uint64_t* d_offsets, uint32_t num_offsets,
                        hipStream_t stream);
hipError_t launch_upload_words(const uint64_t* host_words, size_t nwords, uint64_t* dst,
                               hipStream_t stream);
hipError_t launch_build_tile_map(const TensorDesc* table, uint32_t num_tensors,
                                 uint32_t* tile_map, hipStream_t stream);
hipError_t launch_extract(const ExtractArgs& a, bool idx64, hipStream_t stream);

hipError_t launch_apply(uint16_t* w, uint64_t n, bool idx64, const void* idx,
                        const uint16_t* val, uint64_t count, uint32_t* err,
                        hipStream_t stream);
hipError_t launch_apply_multi(const uint64_t* bases, uint16_t* const* ptrs, uint32_t T,
                              const int64_t* idx, const uint16_t* val, uint64_t count,
                              uint32_t* err, hipStream_t stream);

// Thread-local detail text behind delta_last_error() (abi.hip).
void set_error(const char* fmt, ...) __attribute__((format(printf, 1, 2)));
void clear_error();

}  // namespace aurora
