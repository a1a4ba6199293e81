// Internal interface between the host entry points (adaserve.cpp) and the
// gfx950 kernels (*.hip).  Not part of the public ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace adaserve {

struct TreeAttnArgs {
  const int32_t *node_indptr;  // [B+1]
  const int32_t *parent;       // [T] local ids
  const int32_t *prefix_len;   // [B]
  const int32_t *block_table;  // [B, bt_stride]
  int32_t bt_stride;
  int32_t num_pages;
  const void *q;               // [T, Hq, D]
  const void *k_tree;          // [T, Hkv, D]
  const void *v_tree;
  const void *k_pages;         // [num_pages, Hkv, 16, D]
  const void *v_pages;
  void *out;                   // [T, Hq, D]
  float *ws_o;                 // [units, kRowsPerTile, D] partial numerators
  float *ws_ml;                // [units, kRowsPerTile, 2]  (running max in log2 units, denominator)
  int32_t num_requests;
  int32_t total_nodes;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t group;               // Hq / Hkv
  int32_t chunk_keys;          // prefix keys per unit (multiple of the key block)
  int64_t units;               // work units in the batch
  int64_t padded_grid;         // units rounded up to the XCD count
  int64_t row_groups;          // sum over requests of Hkv * row tiles
  float sm_scale;
  float scale_log2;            // sm_scale * log2(e)
};

hipError_t launch_tree_attn_bf16(const TreeAttnArgs &a, int head_dim, bool needs_combine,
                                 hipStream_t stream);
hipError_t launch_tree_attn_f32(const TreeAttnArgs &a, int head_dim, hipStream_t stream);

hipError_t launch_node_argmax(const void *logits, int64_t row_stride, int32_t rows, int32_t vocab,
                              bool bf16, int32_t *out, hipStream_t stream);

hipError_t launch_tree_accept(int32_t num_requests, int32_t total_nodes, const int32_t *indptr,
                              const int32_t *parent, const int32_t *draft, const int32_t *amax,
                              int32_t max_accept, int32_t *accept_len, int32_t *accept_tokens,
                              int32_t *accept_nodes, hipStream_t stream);

}  // namespace adaserve
