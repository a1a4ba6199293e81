// Host-only part of the library: argument validation and the split-KV work
// planner of the tree-attention entry points.  Plain C++17 with no HIP
// dependency, so it can be built and checked on its own (the CPU sanitizer
// build compiles this file with g++ -fsanitize=address,undefined).
#pragma once
#include <stddef.h>
#include <stdint.h>

#include <utility>
#include <vector>

#include "adaserve.h"
#include "plan.h"

namespace adaserve {

// Records a printf-style message for adaserve_last_error() on this thread and
// returns `code`.
int32_t fail(int32_t code, const char *fmt, ...);
const char *last_error_message();

struct AttnShape {
  int32_t num_requests = 0;
  int32_t total_nodes = 0;
  int32_t group = 0;
};

// Scalar and host-mirror validation shared by the workspace query and the
// verify calls.  bt_stride_or_neg < 0 skips the block-table width check.
int32_t validate_attn_shape(int32_t num_requests, const int32_t *indptr_host, const int32_t *plen_host,
                            int32_t hq, int32_t hkv, int32_t head_dim, int32_t page_size, int32_t dtype,
                            int32_t bt_stride_or_neg, AttnShape &shape);

struct AttnPlan {
  int32_t rows_per_tile = 0;
  int32_t chunk_target = 0;
  int32_t chunk_floor = 0;
  std::vector<int32_t> chunk_len;  // prefix keys per unit of each request
  int64_t units = 0;
  int64_t padded_grid = 0;
  int64_t row_groups = 0;
  bool needs_combine = false;
  bool single_tile = false;        // every request fits one row tile: each K/V byte is read by one unit
  size_t ws_o_bytes = 0;
  size_t ws_ml_bytes = 0;
  size_t ws_bytes = 0;
  double est_us = 0.0;
};

size_t round_up(size_t x, size_t a);

// Makespan of units dealt longest first onto the resident workgroup slots;
// `units` holds (duration, count) pairs and is sorted in place.
double lpt_makespan(std::vector<std::pair<double, int64_t>> &units);

// Work plan of the bf16 kernel for a validated batch (host sizes only); an
// empty plan (no units) for F32 or an empty batch.
AttnPlan make_plan(int32_t B, const int32_t *indptr_host, const int32_t *plen_host, int32_t hkv,
                   int32_t group, int32_t head_dim, int32_t dtype);

// make_plan through a one-entry cache per thread, keyed by the scalar
// arguments and the contents of both host mirrors (not their addresses: a
// caller may refill the same buffers between calls).  The workspace query
// and the verify call of one batch then plan it once, and a batch verified
// again (a retried or repeated step) costs a comparison of 2B + 1 integers.
AttnPlan make_plan_cached(int32_t B, const int32_t *indptr_host, const int32_t *plen_host, int32_t hkv,
                          int32_t group, int32_t head_dim, int32_t dtype);

// The dispatch-ordered request table for batches of at most kPlanMax
// requests (count = 0 otherwise).
struct PlanTable {
  int32_t count = 0;
  int64_t merge_blocks = 0;   // 16-row split-KV merge workgroups of the split requests
  PlanEntry entry[kPlanMax];
};
void fill_plan_table(PlanTable &t, int32_t B, const int32_t *indptr_host, const int32_t *plen_host,
                     int32_t num_kv_heads, int32_t group, const AttnPlan &p);

}  // namespace adaserve
