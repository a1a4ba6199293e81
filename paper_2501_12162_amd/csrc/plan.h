// Work decomposition of the paged tree-attention kernel.
//
// One work unit = (request r, kv-head g, row tile, prefix chunk).  The rows
// of (r, g) are the N_r * G (node, q-head-in-group) pairs, row m = node *
// G + head-in-group, cut into tiles of `rows_per_tile` rows (64 or 128).
// The prefix of r is cut into chunks of whole 32-key blocks, at most
// kMaxChunk keys each: the chunk length of each request comes from the plan
// table in the kernel arguments, or, for batches too large for the table,
// from chunk_keys() below.  A request with an empty prefix still has one
// (empty) chunk.  The last chunk of every (r, g, tile) also takes the
// request's tree block, so every row sees each visible key exactly once.
//
// A split prefix costs partial results: per unit, rows * (2 D + 8) bytes
// (a bf16 output row, an fp32 max and denominator) written and read back
// against chunk * D * 4 bytes of bf16 K and V streamed, i.e. a traffic
// ratio of about rows / chunk.  chunk_keys() therefore never goes below
// `floor_mult` * rows keys (the planner picks 8, 16 or 32); above that
// floor the batch-wide `chunk_target` sets the split.
//
// Units are numbered request by request; inside a request the order is
// (chunk, g, tile) with the tile fastest, so the tiles that read the same KV
// chunk are neighbours (and mostly land on one XCD, see xcd_swizzle), and
// the runs of units an XCD takes spread over every kv-head.
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
                               int32_t chunk_target, int32_t floor_mult) {
  const int32_t rows = n_nodes * group < rows_per_tile ? n_nodes * group : rows_per_tile;
  int32_t c = kMinChunk;
  while (c < floor_mult * rows && c < kMaxChunk) c *= 2;
  return c > chunk_target ? c : chunk_target;
}

ADASERVE_HD int32_t prefix_chunks(int32_t prefix_len, int32_t chunk) {
  return prefix_len > 0 ? ceil_div(prefix_len, chunk) : 1;
}

ADASERVE_HD int64_t request_units(int32_t n_nodes, int32_t prefix_len, int32_t num_kv_heads,
                                  int32_t group, int32_t rows_per_tile, int32_t chunk_target,
                                  int32_t floor_mult) {
  return (int64_t)num_kv_heads * row_tiles(n_nodes, group, rows_per_tile) *
         prefix_chunks(prefix_len, chunk_keys(n_nodes, group, rows_per_tile, chunk_target, floor_mult));
}

// Requests in descending order of per-unit cost, carried in the kernel
// arguments so a workgroup finds its unit without touching memory.  Batches
// with more requests fall back to a scan of node_indptr / prefix_len.
constexpr int kPlanMax = 160;
struct PlanEntry {
  int32_t unit_end;   // exclusive end of this request's units in dispatch order
  int32_t group_end;  // exclusive end of its 16-row merge blocks, same order (none when unsplit)
  int32_t request_and_chunk;  // request (bits 0..15) | prefix keys per unit / 32 << 16
  int32_t node_base;  // node_indptr[request]
  int32_t n_and_len;  // tree nodes (bits 0..7) | prefix length << 8
};

// Field packing of a plan entry: request < kPlanMax, blocks per chunk <=
// kMaxChunk / 32, tree nodes <= kMaxTreeNodes, prefix length < 2^23 (the
// host validation's limit), so every field fits its bits.
ADASERVE_HD int32_t pack_request_chunk(int32_t request, int32_t chunk_blocks) {
  return (int32_t)((uint32_t)request | ((uint32_t)chunk_blocks << 16));
}
ADASERVE_HD int32_t plan_request(int32_t v) { return v & 0xffff; }
ADASERVE_HD int32_t plan_chunk_keys(int32_t v) { return (int32_t)((uint32_t)v >> 16) * kKeysPerBlock; }
ADASERVE_HD int32_t pack_nodes_len(int32_t n, int32_t len) {
  return (int32_t)((uint32_t)n | ((uint32_t)len << 8));
}
ADASERVE_HD int32_t plan_nodes(int32_t v) { return v & 0xff; }
ADASERVE_HD int32_t plan_prefix_len(int32_t v) { return (int32_t)((uint32_t)v >> 8); }
constexpr int32_t kMaxPrefixLen = (1 << 23) - 1;

// Workgroup id -> logical unit id.  Hardware deals consecutive workgroup ids
// to the XCDs round-robin.  Logical units are grouped in runs of kXcdRun
// consecutive ids, and each round of kXcds runs is dealt one run per XCD,
// in XCD order on even rounds and in reverse on odd ones.  Neighbouring
// units (the row tiles that read the same KV chunk) therefore share an L2,
// every XCD takes its runs from the same moving window of the dispatch
// order (the longest-first order is kept chip-wide), and since the order is
// longest first, the reversal keeps the heaviest run of every round from
// landing on the same XCD (mixed-slo attention 6% faster than plain
// round-robin).  The grid must be padded to a multiple of kXcds * kXcdRun;
// ids past `units` do nothing.
constexpr int kXcdRun = 8;

ADASERVE_HD int64_t xcd_swizzle(int64_t block, int64_t padded_grid) {
  (void)padded_grid;
  const int64_t x = block % kXcds, j = block / kXcds;
  const int64_t round = j / kXcdRun;
  const int64_t xs = (round & 1) ? kXcds - 1 - x : x;
  return round * (kXcds * kXcdRun) + xs * kXcdRun + (j % kXcdRun);
}

ADASERVE_HD int64_t pad_to_xcds(int64_t n) {
  const int64_t q = (int64_t)kXcds * kXcdRun;
  return ((n + q - 1) / q) * q;
}

}  // namespace adaserve
