// Work decomposition of the paged tree-attention kernel.
//
// One work unit = (request r, kv-head g, row tile, prefix chunk).  The rows
// of (r, g) are the N_r * G (node, q-head-in-group) pairs, row m = node *
// G + head-in-group, cut into tiles of `rows_per_tile` rows (64 or 128).
// The prefix of r is cut into chunks of chunk_keys(r) keys; a request with
// an empty prefix still has one (empty) chunk.  The last chunk of every
// (r, g, tile) also takes the request's tree block, so every row sees each
// visible key exactly once.
//
// A split prefix costs fp32 partial results: per unit, rows * D * 4 bytes
// written and read back against chunk * D * 4 bytes of bf16 K and V
// streamed, i.e. a traffic ratio of about 2 * rows / chunk.  chunk_keys()
// therefore never goes below 32 * rows (ratio <= 1/16); above that floor the
// batch-wide `chunk_target` sets the split.
//
// Units are numbered request by request; inside a request the order is
// (g, chunk, tile) with the tile fastest, so the tiles that read the same KV
// chunk are neighbours (and land on one XCD, see xcd_swizzle).
//
// The host planner and the device-side unit lookup both use the functions
// below, so their arithmetic cannot drift apart.
#pragma once
#include <stdint.h>

#ifndef __HIPCC__
#define ADASERVE_HD inline
#else
#define ADASERVE_HD __host__ __device__ inline
#endif

namespace adaserve {

constexpr int kMaxRowsPerTile = 128;  // 4 waves x 32 rows
constexpr int kKeysPerBlock = 32;     // keys per LDS pipeline stage
constexpr int kPageSize = 16;
constexpr int kMaxTreeNodes = 128;
constexpr int kMinChunk = 256;
constexpr int kMaxChunk = 8192;       // prefix keys per unit (512 pages)
constexpr int kXcds = 8;              // MI355X: 8 XCDs, workgroups dealt round-robin

ADASERVE_HD int32_t ceil_div(int32_t a, int32_t b) { return (a + b - 1) / b; }

ADASERVE_HD int32_t row_tiles(int32_t n_nodes, int32_t group, int32_t rows_per_tile) {
  return ceil_div(n_nodes * group, rows_per_tile);
}

// Prefix keys per unit for a request with n_nodes tree nodes.
ADASERVE_HD int32_t chunk_keys(int32_t n_nodes, int32_t group, int32_t rows_per_tile,
                               int32_t chunk_target) {
  const int32_t rows = n_nodes * group < rows_per_tile ? n_nodes * group : rows_per_tile;
  int32_t c = kMinChunk;
  while (c < 32 * rows && c < kMaxChunk) c *= 2;
  return c > chunk_target ? c : chunk_target;
}

ADASERVE_HD int32_t prefix_chunks(int32_t prefix_len, int32_t chunk) {
  return prefix_len > 0 ? ceil_div(prefix_len, chunk) : 1;
}

ADASERVE_HD int64_t request_units(int32_t n_nodes, int32_t prefix_len, int32_t num_kv_heads,
                                  int32_t group, int32_t rows_per_tile, int32_t chunk_target) {
  return (int64_t)num_kv_heads * row_tiles(n_nodes, group, rows_per_tile) *
         prefix_chunks(prefix_len, chunk_keys(n_nodes, group, rows_per_tile, chunk_target));
}

// Workgroup id -> logical unit id.  Hardware deals consecutive workgroup ids
// to the XCDs round-robin; this sends logical units u, u+1, ... to one XCD so
// neighbouring units (same KV chunk, different row tiles) share an L2.  The
// grid must be padded to a multiple of kXcds; ids past `units` do nothing.
ADASERVE_HD int64_t xcd_swizzle(int64_t block, int64_t padded_grid) {
  const int64_t per_xcd = padded_grid / kXcds;
  return (block % kXcds) * per_xcd + block / kXcds;
}

ADASERVE_HD int64_t pad_to_xcds(int64_t n) { return ((n + kXcds - 1) / kXcds) * kXcds; }

}  // namespace adaserve
