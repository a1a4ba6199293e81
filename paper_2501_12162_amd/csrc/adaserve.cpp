// Host side of the C ABI declared in include/adaserve.h: argument
// validation (pure host code, runs before any HIP call), the split-KV work
// planner, the gfx950 device check and the kernel launches.
#include "adaserve.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <algorithm>
#include <iterator>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "host_plan.h"
#include "kernels.h"
#include "plan.h"

namespace {

using namespace adaserve;

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

// gfx950 check, once per device ordinal.
int32_t check_device() {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(ADASERVE_ERR_DEVICE, "hipGetDevice failed: %s", hipGetErrorString(e));
  static std::mutex mu;
  static signed char arch_ok[256];  // 0 unknown, 1 gfx950, -1 other
  if (dev < 0 || dev >= 256) return fail(ADASERVE_ERR_DEVICE, "device ordinal %d out of range", dev);
  std::lock_guard<std::mutex> lock(mu);
  if (arch_ok[dev] == 0) {
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess)
      return fail(ADASERVE_ERR_DEVICE, "hipGetDeviceProperties failed: %s", hipGetErrorString(e));
    arch_ok[dev] = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : -1;
  }
  if (arch_ok[dev] < 0) return fail(ADASERVE_ERR_UNSUPPORTED, "device %d is not gfx950", dev);
  return ADASERVE_OK;
}

int32_t launch_status(hipError_t e, const char *what) {
  if (e == hipSuccess) return ADASERVE_OK;
  return fail(ADASERVE_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

}  // namespace

// Beam step: scalar validation shared by the workspace query and the call.
// On success `parts` is the number of scan workgroups per row and `bytes`
// the workspace size ((max, sum) pairs, then the per-part sorted lists).
int32_t validate_beam_shape(int32_t num_requests, int32_t beam_in, int32_t vocab, int32_t beam_out,
                            int32_t dtype, int32_t &parts, size_t &bytes) {
  if (num_requests < 0) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "num_requests %d < 0", num_requests);
  if (beam_in < 1 || beam_in > kBeamMaxWidth)
    return fail(beam_in < 1 ? ADASERVE_ERR_INVALID_ARGUMENT : ADASERVE_ERR_UNSUPPORTED,
                "beam_in %d outside [1, %d]", beam_in, kBeamMaxWidth);
  if (beam_out < 1 || beam_out > kBeamMaxWidth)
    return fail(beam_out < 1 ? ADASERVE_ERR_INVALID_ARGUMENT : ADASERVE_ERR_UNSUPPORTED,
                "beam_out %d outside [1, %d]", beam_out, kBeamMaxWidth);
  if (vocab < 1 || vocab > kBeamMaxVocab)
    return fail(vocab < 1 ? ADASERVE_ERR_INVALID_ARGUMENT : ADASERVE_ERR_UNSUPPORTED, "vocab %d outside [1, %d]",
                vocab, kBeamMaxVocab);
  if (dtype != ADASERVE_F32 && dtype != ADASERVE_BF16)
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "dtype %d is neither F32 nor BF16", dtype);
  parts = beam_parts(vocab, dtype == ADASERVE_BF16);
  const int64_t rows = (int64_t)num_requests * beam_in;
  if (rows * parts > INT32_MAX || (int64_t)num_requests * beam_out > INT32_MAX)
    return fail(ADASERVE_ERR_UNSUPPORTED, "%lld logit rows of %d entries exceed the launch limit", (long long)rows,
                vocab);
  bytes = rows == 0 ? 0 : round_up((size_t)(rows * parts) * 8, 256) + (size_t)(rows * parts) * beam_out * 8;
  return ADASERVE_OK;
}

extern "C" {

const char *adaserve_last_error(void) { return last_error_message(); }

size_t adaserve_tree_attn_workspace_bytes(int32_t num_requests, const int32_t *node_indptr_host,
                                          const int32_t *prefix_len_host, int32_t num_q_heads,
                                          int32_t num_kv_heads, int32_t head_dim, int32_t page_size,
                                          int32_t dtype) {
  AttnShape shape;
  if (validate_attn_shape(num_requests, node_indptr_host, prefix_len_host, num_q_heads, num_kv_heads,
                          head_dim, page_size, dtype, -1, shape) != ADASERVE_OK)
    return SIZE_MAX;
  return make_plan_cached(num_requests, node_indptr_host, prefix_len_host, num_kv_heads, shape.group, head_dim, dtype)
      .ws_bytes;
}

}  // extern "C"

namespace {

// The argmax and acceptance arguments of the whole verification step.
struct StepArgs {
  const void *logits;
  int64_t row_stride;
  int32_t vocab;
  const int32_t *draft_tokens;
  int32_t max_accept;
  int32_t *target_argmax;
  int32_t *accept_len;
  int32_t *accept_tokens;
  int32_t *accept_nodes;
};

// Host checks of the step's argmax and acceptance arguments (the attention
// arguments are checked by tree_attn_verify_impl).
int32_t validate_step(const StepArgs &st, int32_t num_requests, int32_t total_nodes, int32_t dtype) {
  if (st.max_accept < 1) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "max_accept %d < 1", st.max_accept);
  if ((int64_t)num_requests * st.max_accept > INT32_MAX)
    return fail(ADASERVE_ERR_UNSUPPORTED, "num_requests * max_accept exceeds 2^31 - 1");
  if (st.vocab < 1) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "vocab %d < 1", st.vocab);
  if (st.row_stride < st.vocab)
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "row_stride %lld < vocab %d", (long long)st.row_stride, st.vocab);
  if (num_requests == 0) return ADASERVE_OK;
  if (!st.accept_len || !st.accept_tokens || !st.accept_nodes || !st.target_argmax)
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "a required device pointer is NULL");
  if (total_nodes > 0 && (!st.logits || !st.draft_tokens))
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "a required device pointer is NULL");
  const size_t esz = dtype == ADASERVE_BF16 ? 2 : 4;
  if (!aligned(st.logits, esz) || !aligned(st.target_argmax, 4))
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "misaligned logits or argmax pointer");
  return ADASERVE_OK;
}

// The tree-attention entry points and the verification step: the caller's
// workspace, or (use_scratch) the library's static per-device scratch array;
// with `step`, the argmax and acceptance of the same pass are enqueued too.
int32_t tree_attn_verify_impl(int32_t num_requests, const int32_t *node_indptr, const int32_t *node_indptr_host,
                              const int32_t *parent, const void *q, const void *k_tree, const void *v_tree,
                              const void *k_pages, const void *v_pages, int32_t num_pages,
                              const int32_t *block_table, int32_t block_table_stride, const int32_t *prefix_len,
                              const int32_t *prefix_len_host, int32_t num_q_heads, int32_t num_kv_heads,
                              int32_t head_dim, int32_t page_size, float sm_scale, int32_t dtype, void *out,
                              void *workspace, size_t workspace_bytes, bool use_scratch, const StepArgs *step,
                              void *stream) {
  if (block_table_stride < 0) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "block_table_stride < 0");
  if (num_pages < 0) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "num_pages < 0");
  if (!std::isfinite(sm_scale)) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "sm_scale is not finite");
  AttnShape shape;
  int32_t st = validate_attn_shape(num_requests, node_indptr_host, prefix_len_host, num_q_heads, num_kv_heads,
                                   head_dim, page_size, dtype, block_table_stride, shape);
  if (st != ADASERVE_OK) return st;
  // the bf16 kernel's online softmax takes the running maximum of the scaled
  // scores in raw units, which orders them only for a positive scale
  if (dtype == ADASERVE_BF16 && !(sm_scale > 0.f))
    return fail(ADASERVE_ERR_UNSUPPORTED, "sm_scale %g: the BF16 path needs sm_scale > 0", (double)sm_scale);
  if (step) {
    st = validate_step(*step, num_requests, shape.total_nodes, dtype);
    if (st != ADASERVE_OK) return st;
  }
  if (num_requests == 0) return ADASERVE_OK;
  if (!node_indptr || !parent || !q || !k_tree || !v_tree || !out || !prefix_len)
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "a required device pointer is NULL");
  bool any_prefix = false;
  for (int32_t r = 0; r < num_requests; ++r) any_prefix |= prefix_len_host[r] > 0;
  if (any_prefix) {
    if (!k_pages || !v_pages || !block_table)
      return fail(ADASERVE_ERR_INVALID_ARGUMENT, "k_pages, v_pages and block_table are required when a prefix is non-empty");
    if (num_pages < 1) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "num_pages must be >= 1 when a prefix is non-empty");
  }
  const void *tensors[] = {q, k_tree, v_tree, out, k_pages, v_pages};
  for (const void *t : tensors)
    if (t && !aligned(t, 16)) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "tensor pointers must be 16-byte aligned");
  const AttnPlan plan =
      make_plan_cached(num_requests, node_indptr_host, prefix_len_host, num_kv_heads, shape.group, head_dim, dtype);
  if (use_scratch) {
    if (plan.ws_bytes > (size_t)ADASERVE_TREE_ATTN_SCRATCH_BYTES)
      return fail(ADASERVE_ERR_WORKSPACE,
                  "this batch needs %zu bytes of split-KV scratch; the static scratch holds %zu "
                  "(call adaserve_tree_attn_verify with a workspace instead)",
                  plan.ws_bytes, (size_t)ADASERVE_TREE_ATTN_SCRATCH_BYTES);
  } else if (plan.ws_bytes > 0) {
    if (!workspace || workspace_bytes < plan.ws_bytes)
      return fail(ADASERVE_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", plan.ws_bytes,
                  workspace ? workspace_bytes : (size_t)0);
    if (!aligned(workspace, 256)) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
  }
  st = check_device();
  if (st != ADASERVE_OK) return st;
  if (use_scratch && plan.ws_bytes > 0) {
    const hipError_t e = tree_attn_scratch(&workspace);
    if (e != hipSuccess) return launch_status(e, "scratch address lookup");
  }

  TreeAttnArgs a{};
  a.node_indptr = node_indptr;
  a.parent = parent;
  a.prefix_len = prefix_len;
  a.block_table = block_table;
  a.bt_stride = block_table_stride;
  a.num_pages = num_pages;
  a.q = q;
  a.k_tree = k_tree;
  a.v_tree = v_tree;
  a.k_pages = k_pages;
  a.v_pages = v_pages;
  a.out = out;
  a.ws_o = plan.ws_bytes ? (__bf16 *)workspace : nullptr;
  a.ws_ml = plan.ws_bytes ? (float *)((char *)workspace + plan.ws_o_bytes) : nullptr;
  a.num_requests = num_requests;
  a.total_nodes = shape.total_nodes;
  a.num_q_heads = num_q_heads;
  a.num_kv_heads = num_kv_heads;
  a.group = shape.group;
  a.rows_per_tile = plan.rows_per_tile;
  a.chunk_target = plan.chunk_target;
  a.chunk_floor = plan.chunk_floor;
  a.units = plan.units;
  a.padded_grid = plan.padded_grid;
  a.row_groups = plan.row_groups;
  a.merge_blocks = plan.row_groups * (kMaxRowsPerTile / 16);
  a.stream_kv = plan.single_tile ? 1 : 0;
  if (dtype == ADASERVE_BF16) {
    PlanTable t;
    fill_plan_table(t, num_requests, node_indptr_host, prefix_len_host, num_kv_heads, shape.group, plan);
    a.plan_count = t.count;
    if (t.count > 0) {
      std::copy(t.entry, t.entry + t.count, a.plan);
      a.merge_blocks = t.merge_blocks;
    }
  }
  a.sm_scale = sm_scale;
  a.scale_log2 = sm_scale * 1.4426950408889634f;
  hipStream_t s = (hipStream_t)stream;
  if (step && dtype == ADASERVE_BF16) {
    a.logits = step->logits;
    a.logit_stride = step->row_stride;
    a.vocab = step->vocab;
    a.argmax_rows = shape.total_nodes;
    a.argmax_out = step->target_argmax;
    a.draft_tokens = step->draft_tokens;
    a.max_accept = step->max_accept;
    a.accept_requests = num_requests;
    a.accept_len = step->accept_len;
    a.accept_tokens = step->accept_tokens;
    a.accept_nodes = step->accept_nodes;
    return launch_status(launch_verify_step_bf16(a, head_dim, plan.needs_combine, s), "verification step launch");
  }
  if (dtype == ADASERVE_BF16) {
    st = launch_status(launch_tree_attn_bf16(a, head_dim, plan.needs_combine, s), "tree attention launch");
  } else {
    st = launch_status(launch_tree_attn_f32(a, head_dim, s), "tree attention launch");
  }
  if (st != ADASERVE_OK || !step) return st;
  st = launch_status(launch_node_argmax(step->logits, step->row_stride, shape.total_nodes, step->vocab,
                                        dtype == ADASERVE_BF16, step->target_argmax, s),
                     "argmax launch");
  if (st != ADASERVE_OK) return st;
  return launch_status(launch_tree_accept(num_requests, shape.total_nodes, node_indptr, parent, step->draft_tokens,
                                          step->target_argmax, step->max_accept, step->accept_len,
                                          step->accept_tokens, step->accept_nodes, s),
                       "accept launch");
}

}  // namespace

extern "C" {

int32_t adaserve_tree_attn_verify(int32_t num_requests, const int32_t *node_indptr,
                                  const int32_t *node_indptr_host, const int32_t *parent, const void *q,
                                  const void *k_tree, const void *v_tree, const void *k_pages,
                                  const void *v_pages, int32_t num_pages, const int32_t *block_table,
                                  int32_t block_table_stride, const int32_t *prefix_len,
                                  const int32_t *prefix_len_host, int32_t num_q_heads, int32_t num_kv_heads,
                                  int32_t head_dim, int32_t page_size, float sm_scale, int32_t dtype,
                                  void *out, void *workspace, size_t workspace_bytes, void *stream) {
  return tree_attn_verify_impl(num_requests, node_indptr, node_indptr_host, parent, q, k_tree, v_tree, k_pages,
                               v_pages, num_pages, block_table, block_table_stride, prefix_len, prefix_len_host,
                               num_q_heads, num_kv_heads, head_dim, page_size, sm_scale, dtype, out, workspace,
                               workspace_bytes, false, nullptr, stream);
}

int32_t adaserve_tree_attn_verify_noalloc(int32_t num_requests, const int32_t *node_indptr,
                                          const int32_t *node_indptr_host, const int32_t *parent, const void *q,
                                          const void *k_tree, const void *v_tree, const void *k_pages,
                                          const void *v_pages, int32_t num_pages, const int32_t *block_table,
                                          int32_t block_table_stride, const int32_t *prefix_len,
                                          const int32_t *prefix_len_host, int32_t num_q_heads,
                                          int32_t num_kv_heads, int32_t head_dim, int32_t page_size,
                                          float sm_scale, int32_t dtype, void *out, void *stream) {
  return tree_attn_verify_impl(num_requests, node_indptr, node_indptr_host, parent, q, k_tree, v_tree, k_pages,
                               v_pages, num_pages, block_table, block_table_stride, prefix_len, prefix_len_host,
                               num_q_heads, num_kv_heads, head_dim, page_size, sm_scale, dtype, out, nullptr, 0,
                               true, nullptr, stream);
}

int32_t adaserve_tree_verify_step(int32_t num_requests, const int32_t *node_indptr, const int32_t *node_indptr_host,
                                  const int32_t *parent, const void *q, const void *k_tree, const void *v_tree,
                                  const void *k_pages, const void *v_pages, int32_t num_pages,
                                  const int32_t *block_table, int32_t block_table_stride, const int32_t *prefix_len,
                                  const int32_t *prefix_len_host, int32_t num_q_heads, int32_t num_kv_heads,
                                  int32_t head_dim, int32_t page_size, float sm_scale, int32_t dtype,
                                  const void *logits, int64_t logits_row_stride, int32_t vocab,
                                  const int32_t *draft_tokens, int32_t max_accept, void *out, int32_t *target_argmax,
                                  int32_t *accept_len, int32_t *accept_tokens, int32_t *accept_nodes,
                                  void *workspace, size_t workspace_bytes, void *stream) {
  const StepArgs step{logits, logits_row_stride, vocab, draft_tokens, max_accept, target_argmax, accept_len,
                      accept_tokens, accept_nodes};
  return tree_attn_verify_impl(num_requests, node_indptr, node_indptr_host, parent, q, k_tree, v_tree, k_pages,
                               v_pages, num_pages, block_table, block_table_stride, prefix_len, prefix_len_host,
                               num_q_heads, num_kv_heads, head_dim, page_size, sm_scale, dtype, out, workspace,
                               workspace_bytes, false, &step, stream);
}

int32_t adaserve_node_argmax(const void *logits, int64_t row_stride, int32_t num_rows, int32_t vocab, int32_t dtype,
                             int32_t *argmax_out, void *stream) {
  if (num_rows < 0) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "num_rows %d < 0", num_rows);
  if (dtype != ADASERVE_F32 && dtype != ADASERVE_BF16) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "unknown dtype %d", dtype);
  if (num_rows == 0) return ADASERVE_OK;
  if (vocab < 1) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "vocab %d < 1", vocab);
  if (row_stride < vocab) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "row_stride %lld < vocab %d", (long long)row_stride, vocab);
  if (!logits || !argmax_out) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "NULL logits or output");
  const size_t esz = dtype == ADASERVE_BF16 ? 2 : 4;
  if (!aligned(logits, esz) || !aligned(argmax_out, 4))
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "misaligned logits or output pointer");
  const int32_t st = check_device();
  if (st != ADASERVE_OK) return st;
  return launch_status(launch_node_argmax(logits, row_stride, num_rows, vocab, dtype == ADASERVE_BF16, argmax_out,
                                          (hipStream_t)stream),
                       "argmax launch");
}

int32_t adaserve_tree_accept(int32_t num_requests, int32_t total_nodes, const int32_t *node_indptr,
                             const int32_t *parent, const int32_t *draft_tokens, const int32_t *target_argmax,
                             int32_t max_accept, int32_t *accept_len, int32_t *accept_tokens, int32_t *accept_nodes,
                             void *stream) {
  if (num_requests < 0) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "num_requests %d < 0", num_requests);
  if (total_nodes < 0) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "total_nodes %d < 0", total_nodes);
  if (max_accept < 1) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "max_accept %d < 1", max_accept);
  if (num_requests == 0) return ADASERVE_OK;
  if (!node_indptr || !accept_len || !accept_tokens || !accept_nodes)
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "a required device pointer is NULL");
  if (total_nodes > 0 && (!parent || !draft_tokens || !target_argmax))
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "a required device pointer is NULL");
  const int32_t st = check_device();
  if (st != ADASERVE_OK) return st;
  return launch_status(launch_tree_accept(num_requests, total_nodes, node_indptr, parent, draft_tokens, target_argmax,
                                          max_accept, accept_len, accept_tokens, accept_nodes, (hipStream_t)stream),
                       "accept launch");
}

int32_t adaserve_commit_accepted_kv(int32_t num_requests, const int32_t *node_indptr, const int32_t *accept_len,
                                    const int32_t *accept_nodes, int32_t max_accept, const void *k_tree,
                                    const void *v_tree, void *k_pages, void *v_pages, int32_t num_pages,
                                    const int32_t *block_table, int32_t block_table_stride,
                                    const int32_t *prefix_len, int32_t num_kv_heads, int32_t head_dim,
                                    int32_t page_size, int32_t dtype, int32_t *new_prefix_len, void *stream) {
  if (num_requests < 0) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "num_requests %d < 0", num_requests);
  if (max_accept < 1) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "max_accept %d < 1", max_accept);
  if (num_pages < 0) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "num_pages %d < 0", num_pages);
  if (block_table_stride < 0)
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "block_table_stride %d < 0", block_table_stride);
  if (num_kv_heads < 1) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "num_kv_heads %d < 1", num_kv_heads);
  if (head_dim < 1) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "head_dim %d < 1", head_dim);
  if (page_size < 1) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "page_size %d < 1", page_size);
  if (dtype != ADASERVE_F32 && dtype != ADASERVE_BF16)
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "dtype %d is neither F32 nor BF16", dtype);
  const int64_t row_bytes = (int64_t)head_dim * (dtype == ADASERVE_BF16 ? 2 : 4);
  if (row_bytes % 16 != 0 || row_bytes > (1 << 20))
    return fail(ADASERVE_ERR_UNSUPPORTED, "head_dim * element size = %lld bytes is not a multiple of 16 "
                "(or exceeds 1 MiB)", (long long)row_bytes);
  if (num_requests == 0) return ADASERVE_OK;
  if (!node_indptr || !accept_len || !accept_nodes || !prefix_len || !new_prefix_len)
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "a required device pointer is NULL");
  if (!k_tree || !v_tree || !k_pages || !v_pages || (block_table_stride > 0 && !block_table))
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "a required device pointer is NULL");
  if (!aligned(k_tree, 16) || !aligned(v_tree, 16) || !aligned(k_pages, 16) || !aligned(v_pages, 16))
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "k_tree, v_tree, k_pages and v_pages must be 16-byte aligned");
  const int32_t st = check_device();
  if (st != ADASERVE_OK) return st;
  CommitArgs a;
  a.num_requests = num_requests;
  a.node_indptr = node_indptr;
  a.accept_len = accept_len;
  a.accept_nodes = accept_nodes;
  a.max_accept = max_accept;
  a.k_tree = k_tree;
  a.v_tree = v_tree;
  a.k_pages = k_pages;
  a.v_pages = v_pages;
  a.num_pages = num_pages;
  a.block_table = block_table;
  a.bt_stride = block_table_stride;
  a.prefix_len = prefix_len;
  a.num_kv_heads = num_kv_heads;
  a.row_bytes = (int32_t)row_bytes;
  a.page_size = page_size;
  a.new_prefix_len = new_prefix_len;
  return launch_status(launch_commit_kv(a, (hipStream_t)stream), "commit launch");
}

int32_t adaserve_select_trees(int32_t num_requests, int32_t num_candidates, const int32_t *cand_indptr,
                              const int32_t *cand_parent, const float *cand_prob, const float *need,
                              int32_t budget, int32_t n_max, int32_t max_nodes, int32_t *tree_size,
                              int32_t *tree_parent, int32_t *tree_cand, void *stream) {
  if (num_requests < 0 || num_requests > kSelectMaxRequests)
    return fail(num_requests < 0 ? ADASERVE_ERR_INVALID_ARGUMENT : ADASERVE_ERR_UNSUPPORTED,
                "num_requests %d outside [0, %d]", num_requests, kSelectMaxRequests);
  if (num_candidates < 0 || num_candidates > kSelectMaxCandidates)
    return fail(num_candidates < 0 ? ADASERVE_ERR_INVALID_ARGUMENT : ADASERVE_ERR_UNSUPPORTED,
                "num_candidates %d outside [0, %d]", num_candidates, kSelectMaxCandidates);
  if (budget < 0) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "budget %d < 0", budget);
  if (n_max < 1) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "n_max %d < 1", n_max);
  if (max_nodes < ADASERVE_MAX_TREE_NODES)
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "max_nodes %d < %d", max_nodes, ADASERVE_MAX_TREE_NODES);
  if (num_requests == 0) return ADASERVE_OK;
  if (!cand_indptr || !need || !tree_size || !tree_parent || !tree_cand)
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "a required device pointer is NULL");
  if (num_candidates > 0 && (!cand_parent || !cand_prob))
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "a required device pointer is NULL");
  const int32_t st = check_device();
  if (st != ADASERVE_OK) return st;
  SelectArgs a;
  a.num_requests = num_requests;
  a.num_candidates = num_candidates;
  a.cand_indptr = cand_indptr;
  a.cand_parent = cand_parent;
  a.cand_prob = cand_prob;
  a.need = need;
  a.budget = budget;
  a.n_max = n_max;
  a.max_nodes = max_nodes;
  a.tree_size = tree_size;
  a.tree_parent = tree_parent;
  a.tree_cand = tree_cand;
  return launch_status(launch_select_trees(a, (hipStream_t)stream), "select launch");
}

size_t adaserve_beam_step_workspace_bytes(int32_t num_requests, int32_t beam_in, int32_t vocab, int32_t beam_out,
                                          int32_t dtype) {
  int32_t parts = 0;
  size_t bytes = 0;
  if (validate_beam_shape(num_requests, beam_in, vocab, beam_out, dtype, parts, bytes) != ADASERVE_OK)
    return SIZE_MAX;
  return bytes;
}

int32_t adaserve_beam_step(int32_t num_requests, int32_t beam_in, const void *logits, int64_t row_stride,
                           int32_t vocab, int32_t dtype, const float *beam_logprob, int32_t beam_out,
                           int32_t *out_parent, int32_t *out_token, float *out_logprob, void *workspace,
                           size_t workspace_bytes, void *stream) {
  int32_t parts = 0;
  size_t need = 0;
  const int32_t v = validate_beam_shape(num_requests, beam_in, vocab, beam_out, dtype, parts, need);
  if (v != ADASERVE_OK) return v;
  if (row_stride < vocab)
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "row_stride %lld < vocab %d", (long long)row_stride, vocab);
  if (num_requests == 0) return ADASERVE_OK;
  if (!logits || !beam_logprob || !out_parent || !out_token || !out_logprob)
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "a required device pointer is NULL");
  const int64_t esz = dtype == ADASERVE_BF16 ? 2 : 4;
  if (!aligned(logits, 16) || (row_stride * esz) % 16 != 0)
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "logits must be 16-byte aligned with rows a multiple of 16 bytes apart");
  if (!aligned(beam_logprob, 4) || !aligned(out_parent, 4) || !aligned(out_token, 4) || !aligned(out_logprob, 4))
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "misaligned beam_logprob or output pointer");
  if (!workspace || workspace_bytes < need)
    return fail(ADASERVE_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", workspace ? workspace_bytes : (size_t)0,
                need);
  if (!aligned(workspace, 256)) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
  const int32_t st = check_device();
  if (st != ADASERVE_OK) return st;
  BeamArgs a;
  a.num_requests = num_requests;
  a.beam_in = beam_in;
  a.beam_out = beam_out;
  a.rows = num_requests * beam_in;
  a.vocab = vocab;
  a.parts = parts;
  a.row_stride = row_stride;
  a.logits = logits;
  a.beam_logprob = beam_logprob;
  a.ws_ml = (float2 *)workspace;
  a.ws_top = (uint64_t *)((char *)workspace + round_up((size_t)a.rows * parts * 8, 256));
  a.out_parent = out_parent;
  a.out_token = out_token;
  a.out_logprob = out_logprob;
  return launch_status(launch_beam_step(a, dtype == ADASERVE_BF16, (hipStream_t)stream), "beam step launch");
}

size_t adaserve_tree_accept_sampled_workspace_bytes(int32_t total_nodes) {
  if (total_nodes < 0) {
    fail(ADASERVE_ERR_INVALID_ARGUMENT, "total_nodes %d < 0", total_nodes);
    return SIZE_MAX;
  }
  return (size_t)total_nodes * kSampledMaxRounds * 16;  // the most statistics parts a node can take
}

int32_t adaserve_tree_accept_sampled(int32_t num_requests, int32_t total_nodes, const int32_t *node_indptr,
                                     const int32_t *parent, const int32_t *draft_tokens, const void *target_logits,
                                     const void *draft_logits, int64_t row_stride, int32_t vocab, int32_t dtype,
                                     const float *u_accept, const float *u_bonus, int32_t max_accept,
                                     int32_t *accept_len, int32_t *accept_tokens, int32_t *accept_nodes,
                                     void *workspace, size_t workspace_bytes, void *stream) {
  if (num_requests < 0) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "num_requests %d < 0", num_requests);
  if (total_nodes < 0) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "total_nodes %d < 0", total_nodes);
  if (max_accept < 1) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "max_accept %d < 1", max_accept);
  if (vocab < 1) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "vocab %d < 1", vocab);
  if (row_stride < vocab)
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "row_stride %lld < vocab %d", (long long)row_stride, vocab);
  if (dtype != ADASERVE_F32 && dtype != ADASERVE_BF16)
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "dtype %d is neither F32 nor BF16", dtype);
  if ((int64_t)num_requests * max_accept > INT32_MAX)
    return fail(ADASERVE_ERR_UNSUPPORTED, "num_requests * max_accept exceeds 2^31 - 1");
  if (num_requests == 0) return ADASERVE_OK;
  if (!node_indptr || !accept_len || !accept_tokens || !accept_nodes)
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "a required device pointer is NULL");
  if (total_nodes > 0 && (!parent || !draft_tokens || !target_logits || !draft_logits || !u_accept || !u_bonus))
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "a required device pointer is NULL");
  const int64_t esz = dtype == ADASERVE_BF16 ? 2 : 4;
  if (!aligned(target_logits, 16) || !aligned(draft_logits, 16) || (row_stride * esz) % 16 != 0)
    return fail(ADASERVE_ERR_INVALID_ARGUMENT,
                "logits must be 16-byte aligned with rows a multiple of 16 bytes apart");
  const SampledStatsParts parts = sampled_stats_parts(total_nodes, vocab, dtype == ADASERVE_BF16);
  const size_t need = (size_t)total_nodes * parts.parts * 16;
  if (need > 0 && (!workspace || workspace_bytes < need))
    return fail(ADASERVE_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", workspace ? workspace_bytes : (size_t)0,
                need);
  if (need > 0 && !aligned(workspace, 16)) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "workspace must be 16-byte aligned");
  const int32_t st = check_device();
  if (st != ADASERVE_OK) return st;
  SampledArgs a;
  a.num_requests = num_requests;
  a.total_nodes = total_nodes;
  a.node_indptr = node_indptr;
  a.parent = parent;
  a.draft_tokens = draft_tokens;
  a.target_logits = target_logits;
  a.draft_logits = draft_logits;
  a.row_stride = row_stride;
  a.vocab = vocab;
  a.u_accept = u_accept;
  a.u_bonus = u_bonus;
  a.max_accept = max_accept;
  a.accept_len = accept_len;
  a.accept_tokens = accept_tokens;
  a.accept_nodes = accept_nodes;
  a.stats = (float4 *)workspace;
  a.stats_parts = parts.parts;
  a.stats_sub = parts.sub;
  return launch_status(launch_sampled_accept(a, dtype == ADASERVE_BF16, (hipStream_t)stream), "sampled accept launch");
}

}  // extern "C"
