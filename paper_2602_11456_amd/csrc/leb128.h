// Internal declarations of the gap + LEB128 index coder (leb128.hip), used
// by the C ABI and the chunked pipeline.  Not part of the public ABI.
#pragma once

#include "delta_internal.h"

namespace aurora {

// Segments of an index stream: entries [offs[s], offs[s + 1]) form segment
// s (offs has num + 1 entries, device memory); its first entry is coded
// relative to bases[s].  num == 0: one segment based at base0.
struct LebSegs {
  const uint64_t* offs;
  const uint64_t* bases;
  uint32_t num;
  int64_t base0;
};

// Segments of one encoder tile: the first and the last segment its entries
// fall in, and the first entry of the first.
struct EncTileSegs {
  uint32_t first, last;
  uint64_t lo0;
};

struct EncArgs {
  const int64_t* idx;
  uint64_t count;               // entries, or the most there can be if d_count_in is set
  const uint64_t* d_count_in;   // nullable: the entry count, in device memory
  LebSegs segs;
  uint8_t* out;
  uint64_t capacity;
  uint64_t* d_nbytes;
  uint64_t* seg_byte_offsets;   // nullable, num + 1 entries
  uint32_t* err;                // nullable
  uint32_t* tile_bytes;
  uint64_t* group_excl;
  uint8_t* stage;               // per tile, its staged code
  EncTileSegs* tile_segs;       // per tile (with segments)
};

// A 16 KiB decode tile's first entry and, with segments, the first and the
// last segment of its entries and the first entry of the first.
struct DecTileRec {
  uint64_t e0;
  uint32_t first, last;
  uint64_t lo0;
};

struct DecArgs {
  const uint8_t* in;
  uint64_t nbytes;
  LebSegs segs;
  int64_t* out;
  uint64_t capacity;
  uint64_t* d_count;
  uint32_t* err;                // nullable
  uint32_t* tile_terms;         // numbers ending in each byte tile
  uint64_t* group_excl;         // entries before each group of tiles
  uint32_t* tile_f;             // byte tile holds a segment start
  uint64_t* tile_v;             // segmented sum of the tile's terms
  uint32_t* wave_f;             // the same per wavefront of a tile (4 per tile)
  uint64_t* wave_v;
  // Decode-in-apply (launch_leb128_decode with apply set): instead of
  // writing index k, write val[k] to the word of the tensor list that
  // decoded index names.
  uint16_t* const* ptrs;        // device [num_tensors]
  const uint64_t* tbases;       // device [num_tensors + 1]: first index of each tensor, total
  uint32_t num_tensors;
  const uint16_t* val;          // device [capacity]
  uint64_t* gexcl_v;            // index just before each group of tiles
  DecTileRec* tile_recs;        // per byte tile (dec_recs_kernel)
};

struct EncLayout {
  uint64_t tiles;
  size_t tile_bytes, group_sum, group_excl, tile_segs, stage, total;
};
// Encoder grid for up to `count` entries.
uint32_t enc_grid(uint64_t count, bool count_on_device);
struct DecLayout {
  uint64_t btiles;
  size_t tile_terms, group_sum, group_excl, tile_f, tile_v, wave_f, wave_v, gsum_f, gsum_v,
      gexcl_v, tile_recs, total;
};
EncLayout enc_layout(uint64_t count);
DecLayout dec_layout(uint64_t nbytes);
// Enqueues the encoder; its tables and staging slots live in `ws` at the
// offsets of `L` (enc_layout of a.count).
hipError_t launch_leb128_encode(EncArgs a, char* ws, const EncLayout& L, hipStream_t stream);
// Decodes a.in; writes the indices to a.out, or, with `apply`, applies
// a.val to the tensors a.ptrs (capacity = entries of a.val; a stream with
// another entry count raises a.err).
hipError_t launch_leb128_decode(DecArgs a, const DecLayout& L, char* ws, hipStream_t stream,
                                bool apply = false);

}  // namespace aurora
