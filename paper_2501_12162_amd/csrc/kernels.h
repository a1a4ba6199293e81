// Internal interface between the host entry points (adaserve.cpp) and the
// gfx950 kernels (*.hip).  Not part of the public ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "plan.h"

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
  const void *zero16;          // 16 zero bytes in device memory (source of masked DMA lanes)
  void *out;                   // [T, Hq, D]
  __bf16 *ws_o;                // [units, kMaxRowsPerTile, D] partial outputs (each chunk normalised)
  float *ws_ml;                // [units, kMaxRowsPerTile, 2]  (reference max in raw units, denominator)
  int32_t num_requests;
  int32_t total_nodes;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t group;               // Hq / Hkv
  int32_t rows_per_tile;       // 64 or 128
  int32_t chunk_target;        // batch-wide prefix chunk (chunk_keys() in plan.h), used when
  int32_t chunk_floor;         // minimum chunk in keys per tile row       plan_count == 0
  int64_t units;               // work units in the batch
  int64_t padded_grid;         // units rounded up to the XCD count
  int64_t row_groups;          // sum over requests of Hkv * row tiles
  int64_t merge_blocks;        // workgroups of the split-KV merge
  float sm_scale;
  float scale_log2;            // sm_scale * log2(e)
  // Fused verification step (adaserve_tree_verify_step; zero counts
  // otherwise): argmax_rows argmax workgroups follow the attention grid, and
  // acceptance waves for accept_requests requests follow the merge grid.
  const void *logits;          // [argmax_rows, logit_stride] bf16
  int64_t logit_stride;
  int32_t vocab;
  int32_t argmax_rows;
  int32_t *argmax_out;         // [argmax_rows]
  const int32_t *draft_tokens; // [total_nodes]
  int32_t max_accept;
  int32_t accept_requests;
  int32_t *accept_len;         // [num_requests]
  int32_t *accept_tokens;      // [num_requests, max_accept]
  int32_t *accept_nodes;       // [num_requests, max_accept]
  int32_t stream_kv;           // 1: every request is one row tile (K/V read once; non-temporal loads)
  int32_t plan_count;          // entries used in plan[] (0: scan the device arrays)
  PlanEntry plan[kPlanMax];
};

hipError_t launch_tree_attn_bf16(TreeAttnArgs &a, int head_dim, bool needs_combine, hipStream_t stream);
// The verification step in two launches: attention + argmax workgroups, then
// the split-KV merge (when a prefix is split) + acceptance waves.
hipError_t launch_verify_step_bf16(TreeAttnArgs &a, int head_dim, bool needs_combine, hipStream_t stream);
// Device address of the static split-KV scratch array on the current device
// (ADASERVE_TREE_ATTN_SCRATCH_BYTES bytes, 256-byte aligned); looked up once
// per device.
hipError_t tree_attn_scratch(void **out);
hipError_t launch_tree_attn_f32(const TreeAttnArgs &a, int head_dim, hipStream_t stream);

hipError_t launch_node_argmax(const void *logits, int64_t row_stride, int32_t rows, int32_t vocab,
                              bool bf16, int32_t *out, hipStream_t stream);

hipError_t launch_tree_accept(int32_t num_requests, int32_t total_nodes, const int32_t *indptr,
                              const int32_t *parent, const int32_t *draft, const int32_t *amax,
                              int32_t max_accept, int32_t *accept_len, int32_t *accept_tokens,
                              int32_t *accept_nodes, hipStream_t stream);

struct CommitArgs {
  int32_t num_requests;
  const int32_t *node_indptr;
  const int32_t *accept_len;
  const int32_t *accept_nodes;   // [num_requests, max_accept]
  int32_t max_accept;
  const void *k_tree;
  const void *v_tree;
  void *k_pages;
  void *v_pages;
  int32_t num_pages;
  const int32_t *block_table;
  int32_t bt_stride;
  const int32_t *prefix_len;
  int32_t num_kv_heads;
  int32_t row_bytes;             // head_dim * element size, a multiple of 16
  int32_t page_size;
  int32_t *new_prefix_len;
};

hipError_t launch_commit_kv(const CommitArgs &a, hipStream_t stream);

constexpr int kSelectMaxCandidates = 8192;  // per batch
constexpr int kSelectMaxRequests = 512;
constexpr int kSelectMaxPerRequest = 127;   // trees of at most 128 nodes

struct SelectArgs {
  int32_t num_requests;
  int32_t num_candidates;
  const int32_t *cand_indptr;   // [num_requests + 1]
  const int32_t *cand_parent;   // [num_candidates] local: -1 = child of the root
  const float *cand_prob;       // [num_candidates] path probabilities
  const float *need;            // [num_requests]
  int32_t budget;
  int32_t n_max;
  int32_t max_nodes;            // output row stride, >= 128
  int32_t *tree_size;           // [num_requests]
  int32_t *tree_parent;         // [num_requests, max_nodes]
  int32_t *tree_cand;           // [num_requests, max_nodes]
};

hipError_t launch_select_trees(const SelectArgs &a, hipStream_t stream);

// One beam-search speculation step (beam.hip).
constexpr int kBeamMaxWidth = 64;
constexpr int kBeamMaxVocab = 1 << 20;
constexpr int kBeamMaxParts = 32;   // row parts at kBeamMaxVocab (fp32: 32768 logits per part)

struct BeamArgs {
  int32_t num_requests;
  int32_t beam_in;              // beams per request (rows per request)
  int32_t beam_out;             // children kept per request
  int32_t rows;                 // num_requests * beam_in
  int32_t vocab;
  int32_t parts;                // workgroups per row (beam_parts)
  int64_t row_stride;           // elements between logit rows
  const void *logits;           // [rows, row_stride]
  const float *beam_logprob;    // [rows]
  float2 *ws_ml;                // [rows, parts] (part max, sum of exp(x - max))
  uint64_t *ws_top;             // [rows, parts, beam_out] sorted row keys (logit, token)
  int32_t *out_parent;          // [num_requests, beam_out]
  int32_t *out_token;
  float *out_logprob;
};

int32_t beam_parts(int32_t vocab, bool bf16);
hipError_t launch_beam_step(const BeamArgs &a, bool bf16, hipStream_t stream);

// Tree verification for sampled decoding (sampled.hip).
constexpr int kMaxSampledNodes = 128;

struct SampledArgs {
  int32_t num_requests;
  int32_t total_nodes;
  const int32_t *node_indptr;   // [B + 1]
  const int32_t *parent;        // [T] local ids
  const int32_t *draft_tokens;  // [T]
  const void *target_logits;    // [T, row_stride]
  const void *draft_logits;     // [T, row_stride]
  int64_t row_stride;           // elements
  int32_t vocab;
  const float *u_accept;        // [T]
  const float *u_bonus;         // [T]
  int32_t max_accept;
  int32_t *accept_len;          // [B]
  int32_t *accept_tokens;       // [B, max_accept]
  int32_t *accept_nodes;        // [B, max_accept]
  float4 *stats;                // [total_nodes, stats_parts] workspace: (max_p, sum_p, max_q, sum_q)
  int32_t stats_parts;          // statistics parts (workgroups) per node: rounds * stats_sub
  int32_t stats_sub;            // parts per round
};

// Round layout of a sampled-verification pass over a row of `vocab` logits,
// epv of them per 16-byte vector: the vectors go in groups of
// kSampledGroupVecs, gpr consecutive groups form a round (a contiguous token
// range), at most kSampledMaxRounds of them; the tokens past the last whole
// vector belong to the last round.
constexpr int kSampledGroupVecs = 4096;
constexpr int kSampledMaxRounds = 64;
struct SampledRounds {
  int nvec, ngroups, gpr, nrounds;
  __host__ __device__ SampledRounds(int vocab, int epv) {
    nvec = vocab / epv;
    ngroups = (nvec + kSampledGroupVecs - 1) / kSampledGroupVecs;
    if (ngroups < 1) ngroups = 1;
    gpr = (ngroups + kSampledMaxRounds - 1) / kSampledMaxRounds;
    nrounds = (ngroups + gpr - 1) / gpr;
  }
};

// The statistics pass splits each round of every node's rows into `sub`
// contiguous parts, one workgroup each: enough parts that a small batch
// still puts several workgroups on every compute unit (4096 in all, at most
// 8 per node unless the rounds alone are more), at most kSampledMaxRounds
// per node.
struct SampledStatsParts {
  int32_t parts, sub;
};
inline SampledStatsParts sampled_stats_parts(int64_t total_nodes, int32_t vocab, bool bf16) {
  constexpr int64_t kTargetGroups = 4096, kMaxWanted = 8;
  int64_t want = total_nodes > 0 ? (kTargetGroups + total_nodes - 1) / total_nodes : 1;
  if (want > kMaxWanted) want = kMaxWanted;
  const int32_t nrounds = SampledRounds(vocab, bf16 ? 8 : 4).nrounds;
  int32_t sub = (int32_t)((want + nrounds - 1) / nrounds);
  if (sub * nrounds > kSampledMaxRounds) sub = kSampledMaxRounds / nrounds;
  return {nrounds * sub, sub};
}

hipError_t launch_sampled_accept(const SampledArgs &a, bool bf16, hipStream_t stream);

}  // namespace adaserve
