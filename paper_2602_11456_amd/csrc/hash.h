// Internal declarations of the integrity hash and the artifact layout
// (hash.hip).  Not part of the public ABI.
#pragma once

#include "delta_internal.h"

namespace aurora {

// The header bytes covered by the artifact hash, and where the hash sits.
constexpr uint64_t kArtifactHashedHeader = 80;
constexpr uint64_t kArtifactHashField = 80;
static_assert(sizeof(delta_artifact_header_t) == 128, "artifact header layout");
static_assert(offsetof(delta_artifact_header_t, hash) == kArtifactHashField, "hash field");

// Byte offsets of the artifact's parts: header | tensor table (24 bytes per
// tensor) | index stream | value stream | segment hash table.  The hashed
// payload is [table, hashes).
struct ArtifactLayout {
  uint64_t table, idx, val, hashes, total, num_segments;
};
ArtifactLayout artifact_layout(uint64_t num_tensors, uint64_t count, uint64_t idx_bytes,
                               uint64_t seg_bytes);

hipError_t launch_hash_segments(const uint8_t* data, uint64_t nbytes, uint64_t seg_bytes,
                                uint64_t seed, uint64_t* out, hipStream_t stream);
// Writes the tensor table from device arrays (numels [T], entry offsets
// [T + 1], first index bytes [T] or NULL for 8 bytes per entry) and zeroes
// the alignment padding after the index and value streams.
hipError_t launch_artifact_table(uint8_t* art, const ArtifactLayout& L, const uint64_t* numels,
                                 const uint64_t* offs, const uint64_t* byte_offs, uint32_t T,
                                 uint64_t idx_bytes, uint64_t count, hipStream_t stream);
hipError_t launch_artifact_seal(uint8_t* art, const ArtifactLayout& L,
                                const delta_artifact_header_t& h, hipStream_t stream);
hipError_t launch_artifact_verify(const uint8_t* art, const ArtifactLayout& L, uint64_t seg_bytes,
                                  uint64_t seed, uint64_t* fresh, uint64_t* d_bad,
                                  uint64_t* d_first_bad, uint32_t* d_header_bad,
                                  hipStream_t stream);

}  // namespace aurora
