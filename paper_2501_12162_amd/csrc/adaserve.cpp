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

#include "kernels.h"
#include "plan.h"

namespace {

using namespace adaserve;

thread_local std::string g_last_error;

int32_t fail(int32_t code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

// gfx950 check, once per device ordinal.
int32_t check_device() {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(ADASERVE_ERR_DEVICE, "hipGetDevice failed: %s", hipGetErrorString(e));
  static std::mutex mu;
  static signed char verdict[256];  // 0 unknown, 1 gfx950, -1 other
  if (dev < 0 || dev >= 256) return fail(ADASERVE_ERR_DEVICE, "device ordinal %d out of range", dev);
  std::lock_guard<std::mutex> lock(mu);
  if (verdict[dev] == 0) {
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess)
      return fail(ADASERVE_ERR_DEVICE, "hipGetDeviceProperties failed: %s", hipGetErrorString(e));
    verdict[dev] = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : -1;
    if (verdict[dev] < 0) g_last_error = std::string("unsupported device architecture ") + prop.gcnArchName;
  }
  if (verdict[dev] < 0) return fail(ADASERVE_ERR_UNSUPPORTED, "device %d is not gfx950", dev);
  return ADASERVE_OK;
}

int32_t launch_status(hipError_t e, const char *what) {
  if (e == hipSuccess) return ADASERVE_OK;
  return fail(ADASERVE_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

struct AttnShape {
  int32_t num_requests = 0;
  int32_t total_nodes = 0;
  int32_t group = 0;
};

// Scalar and host-mirror validation shared by the workspace query and the
// verify call.  Does not touch device memory.
int32_t validate_attn_shape(int32_t num_requests, const int32_t *indptr_host, const int32_t *plen_host,
                            int32_t hq, int32_t hkv, int32_t head_dim, int32_t page_size, int32_t dtype,
                            int32_t bt_stride_or_neg, AttnShape &shape) {
  if (num_requests < 0) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "num_requests %d < 0", num_requests);
  if (hq <= 0 || hkv <= 0) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "head counts must be positive (%d, %d)", hq, hkv);
  if (hq % hkv != 0)
    return fail(ADASERVE_ERR_INVALID_ARGUMENT, "num_q_heads %d is not a multiple of num_kv_heads %d", hq, hkv);
  if (hq / hkv > 16) return fail(ADASERVE_ERR_UNSUPPORTED, "head group %d > 16", hq / hkv);
  if (dtype != ADASERVE_F32 && dtype != ADASERVE_BF16) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "unknown dtype %d", dtype);
  if (head_dim != 64 && head_dim != 128) return fail(ADASERVE_ERR_UNSUPPORTED, "head_dim %d (supported: 64, 128)", head_dim);
  if (page_size != kPageSize) return fail(ADASERVE_ERR_UNSUPPORTED, "page_size %d (supported: 16)", page_size);
  shape.num_requests = num_requests;
  shape.group = hq / hkv;
  if (num_requests == 0) return ADASERVE_OK;
  if (!indptr_host || !plen_host) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "host mirrors must not be NULL");
  if (indptr_host[0] != 0) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "node_indptr[0] = %d, expected 0", indptr_host[0]);
  int64_t total = 0;
  for (int32_t r = 0; r < num_requests; ++r) {
    const int64_t n = (int64_t)indptr_host[r + 1] - indptr_host[r];
    if (n < 1) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "request %d has %lld tree nodes (need >= 1)", r, (long long)n);
    if (n > kMaxTreeNodes) return fail(ADASERVE_ERR_UNSUPPORTED, "request %d has %lld tree nodes (max %d)", r, (long long)n, kMaxTreeNodes);
    total += n;
    const int32_t L = plen_host[r];
    if (L < 0) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "prefix_len[%d] = %d < 0", r, L);
    if (L >= (1 << 23)) return fail(ADASERVE_ERR_UNSUPPORTED, "prefix_len[%d] = %d (max %d)", r, L, (1 << 23) - 1);
    if (bt_stride_or_neg >= 0 && ceil_div(L, kPageSize) > bt_stride_or_neg)
      return fail(ADASERVE_ERR_INVALID_ARGUMENT, "prefix_len[%d] = %d needs %d pages > block_table_stride %d", r, L,
                  ceil_div(L, kPageSize), bt_stride_or_neg);
  }
  if (total > INT32_MAX / 16) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "too many tree nodes (%lld)", (long long)total);
  shape.total_nodes = (int32_t)total;
  return ADASERVE_OK;
}

struct AttnPlan {
  int32_t rows_per_tile = 0;
  int32_t chunk_target = 0;
  int32_t chunk_floor = 0;
  std::vector<int32_t> chunk_len;  // prefix keys per unit of each request
  int64_t units = 0;
  int64_t padded_grid = 0;
  int64_t row_groups = 0;
  bool needs_combine = false;
  size_t ws_o_bytes = 0;
  size_t ws_ml_bytes = 0;
  size_t ws_bytes = 0;
  double est_us = 0.0;
};

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Cost model of the bf16 kernel, measured on MI355X: paged K/V streaming
// over the whole chip; one 32-key pipeline step of a workgroup while two
// workgroups share each CU (it hardly depends on the tile's row count: the
// four waves compute their row blocks side by side); the fixed cost of a
// unit (first loads of the block table, queries and K block 0, then the
// output writes); and the latency the combine kernel adds.
constexpr double kChipBytesPerUs = 5.8e6;
constexpr double kBlockUs = 1.0;
constexpr double kUnitFixedUs = 6.0;
constexpr double kCombineUs = 3.0;
constexpr int kCUs = 256;
constexpr int kSlots = 2 * kCUs;  // resident workgroups: two per CU

// Makespan of units dispatched longest first onto kSlots workgroup slots,
// each unit taking the slot that frees up first (how the hardware deals a
// grid whose units come in that order).  Slot loads are kept as runs of
// equal load, so the cost grows with the number of distinct durations, not
// with the number of units.  `units` holds (duration, count) pairs in any
// order; it is sorted in place.
double lpt_makespan(std::vector<std::pair<double, int64_t>> &units) {
  std::sort(units.begin(), units.end(), [](const auto &x, const auto &y) { return x.first > y.first; });
  size_t m = 0;  // merge equal durations
  for (size_t i = 0; i < units.size(); ++i) {
    if (m > 0 && units[m - 1].first == units[i].first)
      units[m - 1].second += units[i].second;
    else
      units[m++] = units[i];
  }
  units.resize(m);
  std::vector<std::pair<double, int64_t>> runs{{0.0, (int64_t)kSlots}};  // (load, slots), ascending
  std::vector<std::pair<double, int64_t>> moved, rest, merged;
  for (const auto &u : units) {
    const double t = u.first;
    int64_t c = u.second;
    const int64_t rounds = c / kSlots;
    if (rounds > 0) {
      for (auto &x : runs) x.first += (double)rounds * t;
      c -= rounds * kSlots;
    }
    if (c == 0) continue;
    // the c least-loaded slots take one more unit each: an ascending prefix
    // of the runs moves up by t, so two ascending lists are merged back
    moved.clear();
    rest.clear();
    for (const auto &x : runs) {
      if (c == 0) {
        rest.push_back(x);
      } else if (x.second <= c) {
        moved.push_back({x.first + t, x.second});
        c -= x.second;
      } else {
        moved.push_back({x.first + t, c});
        rest.push_back({x.first, x.second - c});
        c = 0;
      }
    }
    merged.clear();
    std::merge(rest.begin(), rest.end(), moved.begin(), moved.end(), std::back_inserter(merged));
    runs.clear();
    for (const auto &x : merged) {
      if (!runs.empty() && runs.back().first == x.first)
        runs.back().second += x.second;
      else
        runs.push_back(x);
    }
  }
  return runs.back().first;
}

// Plan for one choice of per-request chunk lengths `ck` (prefix keys per
// unit, whole 32-key blocks, at most kMaxChunk) with 128-row tiles.  The
// cost estimate is the larger of the longest-first makespan of the units
// and the chip-wide streaming time (K/V plus the split partials, at a rate
// scaled by the share of workgroup slots the units fill), plus the combine
// pass when a prefix is split.  evaluate_plan fills everything but
// the makespan and returns the unit list; `bound` is a lower bound of the
// estimate (the makespan replaced by max(longest unit, total / slots)).
AttnPlan evaluate_plan(int32_t B, const int32_t *indptr_host, const int32_t *plen_host, int32_t hkv,
                       int32_t group, int32_t head_dim, int32_t rows_per_tile, const std::vector<int32_t> &ck,
                       std::vector<std::pair<double, int64_t>> &units, double &fixed, double &bound) {
  AttnPlan p;
  p.rows_per_tile = rows_per_tile;
  p.chunk_len = ck;
  const double key_bytes = 4.0 * head_dim;  // bf16 K and V of one key of one kv-head
  double kv_bytes = 0, partial_bytes = 0, total = 0;
  units.clear();
  for (int32_t r = 0; r < B; ++r) {
    const int32_t n = indptr_host[r + 1] - indptr_host[r];
    const int32_t L = plen_host[r];
    const int32_t tiles = row_tiles(n, group, rows_per_tile);
    const int32_t chunks = prefix_chunks(L, ck[r]);
    const int64_t cnt = (int64_t)hkv * tiles * chunks;
    p.units += cnt;
    p.row_groups += (int64_t)hkv * tiles;
    kv_bytes += (double)hkv * tiles * (L + n) * key_bytes;
    if (chunks > 1) {
      p.needs_combine = true;
      partial_bytes += hkv * chunks * n * group * (head_dim * 2.0 + 8.0);
    }
    // every chunk pays the fixed cost; the tree block is spread over them
    const double blocks = ceil_div(std::min(L, ck[r]), 32) + (double)ceil_div(n, 32) / chunks;
    units.push_back({kUnitFixedUs + blocks * kBlockUs, cnt});
    total += units.back().first * cnt;
  }
  double longest = 0;
  for (const auto &u : units) longest = std::max(longest, u.first);
  // the chip streams at full rate only with every workgroup slot busy
  const double occupancy = std::min(1.0, (double)p.units / kSlots);
  const double stream = (kv_bytes + partial_bytes) / (kChipBytesPerUs * occupancy);
  const double combine = p.needs_combine ? kCombineUs + partial_bytes / kChipBytesPerUs : 0.0;
  fixed = combine;
  p.est_us = std::max(stream, 0.0);  // completed with the makespan by make_plan
  bound = std::max({stream, longest, total / kSlots}) + combine;
  p.padded_grid = pad_to_xcds(p.units);
  if (p.needs_combine) {
    p.ws_o_bytes = round_up((size_t)p.units * kMaxRowsPerTile * head_dim * 2, 256);  // bf16
    p.ws_ml_bytes = round_up((size_t)p.units * kMaxRowsPerTile * 2 * sizeof(float), 256);
    p.ws_bytes = p.ws_o_bytes + p.ws_ml_bytes;
  }
  return p;
}

// Work plan of the bf16 kernel, from host-visible sizes only: the cheapest
// estimate over two families of prefix splits, 128-row tiles.  (A 64-row
// tile costs about as much per step as a 128-row one, so it never wins.)
//  * batch-wide chunk targets {256 .. 8192} with chunk floors {8, 16, 32}
//    keys per row (chunk_keys() in plan.h), the only family the device can
//    rebuild without a plan table;
//  * with a plan table, balanced splits: for a target unit count, every
//    request's prefix is cut into the fewest equal runs of whole 32-key
//    blocks no longer than the batch's mean blocks per unit, so the units
//    come out about equally long and fill the workgroup slots evenly.
// Choices that give every request the same chunk lengths as one already
// tried are skipped, and the makespan is only simulated for choices whose
// lower bound can still beat the best estimate so far.  Requests are then
// dispatched in descending order of per-unit cost (fill_plan_table).
AttnPlan make_plan(int32_t B, const int32_t *indptr_host, const int32_t *plen_host, int32_t hkv,
                   int32_t group, int32_t head_dim, int32_t dtype) {
  AttnPlan best;
  if (dtype != ADASERVE_BF16 || B == 0) return best;
  const int32_t rt = kMaxRowsPerTile;
  struct Cand {
    double bound;
    int32_t fm, c;   // batch-wide family (fm = 0: balanced)
    std::vector<int32_t> ck;
  };
  std::vector<Cand> cands;
  std::vector<std::pair<double, int64_t>> units;
  double fixed, bound;
  auto add = [&](int32_t fm, int32_t c, std::vector<int32_t> ck) {
    for (const Cand &x : cands)
      if (x.ck == ck) return;
    evaluate_plan(B, indptr_host, plen_host, hkv, group, head_dim, rt, ck, units, fixed, bound);
    cands.push_back({bound, fm, c, std::move(ck)});
  };
  std::vector<int32_t> ck(B);
  for (int32_t fm : {32, 16, 8})
    for (int32_t c = kMaxChunk; c >= kMinChunk; c /= 2) {
      for (int32_t r = 0; r < B; ++r) ck[r] = chunk_keys(indptr_host[r + 1] - indptr_host[r], group, rt, c, fm);
      add(fm, c, ck);
    }
  if (B <= kPlanMax) {
    int64_t work = 0;   // unit-blocks of the unsplit batch
    for (int32_t r = 0; r < B; ++r)
      work += (int64_t)hkv * row_tiles(indptr_host[r + 1] - indptr_host[r], group, rt) *
              std::max(1, ceil_div(plen_host[r], kKeysPerBlock));
    for (int32_t target : {256, 320, 384, 448, 512, 576, 640, 768, 1024}) {
      const int64_t per_unit = std::max<int64_t>(4, (work + target - 1) / target);
      for (int32_t r = 0; r < B; ++r) {
        const int32_t blocks = ceil_div(std::max(plen_host[r], 0), kKeysPerBlock);
        if (blocks == 0) {
          ck[r] = kMaxChunk;
          continue;
        }
        const int32_t runs = (int32_t)std::max<int64_t>((blocks + per_unit - 1) / per_unit,
                                                        ceil_div(blocks, kMaxChunk / kKeysPerBlock));
        ck[r] = ceil_div(blocks, runs) * kKeysPerBlock;
      }
      add(0, 0, ck);
    }
  }
  // candidates in the order they were generated break ties (larger chunks first)
  std::stable_sort(cands.begin(), cands.end(), [](const Cand &x, const Cand &y) { return x.bound < y.bound; });
  bool have = false;
  for (const Cand &cd : cands) {
    if (have && cd.bound >= best.est_us * 0.98) break;
    AttnPlan p = evaluate_plan(B, indptr_host, plen_host, hkv, group, head_dim, rt, cd.ck, units, fixed, bound);
    p.est_us = std::max(p.est_us, lpt_makespan(units)) + fixed;
    // the batch-wide fields rebuild the chunks when there is no plan table
    p.chunk_target = cd.fm ? cd.c : kMaxChunk;
    p.chunk_floor = cd.fm ? cd.fm : 32;
    if (!have || p.est_us < best.est_us * 0.98) {
      best = std::move(p);
      have = true;
    }
  }
  return best;
}

// Fills the dispatch-ordered request table (descending per-unit cost) when
// the batch fits in the kernel arguments; otherwise leaves it empty.
void fill_plan_table(TreeAttnArgs &a, int32_t B, const int32_t *indptr_host, const int32_t *plen_host,
                     const AttnPlan &p) {
  a.plan_count = 0;
  if (B > kPlanMax) return;
  int32_t order[kPlanMax];
  int64_t cost[kPlanMax];
  for (int32_t r = 0; r < B; ++r) {
    const int32_t n = indptr_host[r + 1] - indptr_host[r];
    const int32_t keys = std::min(std::max(plen_host[r], 0), p.chunk_len[r]);
    cost[r] = keys + n;  // steps per unit (the step time hardly depends on the row count)
    order[r] = r;
  }
  std::stable_sort(order, order + B, [&](int32_t x, int32_t y) { return cost[x] > cost[y]; });
  int64_t end = 0, gend = 0;
  for (int32_t i = 0; i < B; ++i) {
    const int32_t r = order[i];
    const int32_t n = indptr_host[r + 1] - indptr_host[r];
    end += (int64_t)a.num_kv_heads * row_tiles(n, a.group, p.rows_per_tile) *
           prefix_chunks(plen_host[r], p.chunk_len[r]);
    // merge blocks: 16 rows of one kv-head each, for split requests only
    if (prefix_chunks(plen_host[r], p.chunk_len[r]) > 1) gend += (int64_t)a.num_kv_heads * ceil_div(n * a.group, 16);
    a.plan[i].unit_end = (int32_t)end;
    a.plan[i].group_end = (int32_t)gend;
    a.plan[i].request_and_chunk = r | ((p.chunk_len[r] / kKeysPerBlock) << 16);
    a.plan[i].node_base = indptr_host[r];
    a.plan[i].n_and_len = n | (plen_host[r] << 8);
  }
  a.plan_count = B;
  a.merge_blocks = gend;
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

const char *adaserve_last_error(void) { return g_last_error.c_str(); }

size_t adaserve_tree_attn_workspace_bytes(int32_t num_requests, const int32_t *node_indptr_host,
                                          const int32_t *prefix_len_host, int32_t num_q_heads,
                                          int32_t num_kv_heads, int32_t head_dim, int32_t page_size,
                                          int32_t dtype) {
  AttnShape shape;
  if (validate_attn_shape(num_requests, node_indptr_host, prefix_len_host, num_q_heads, num_kv_heads,
                          head_dim, page_size, dtype, -1, shape) != ADASERVE_OK)
    return SIZE_MAX;
  return make_plan(num_requests, node_indptr_host, prefix_len_host, num_kv_heads, shape.group, head_dim, dtype)
      .ws_bytes;
}

int32_t adaserve_tree_attn_verify(int32_t num_requests, const int32_t *node_indptr,
                                  const int32_t *node_indptr_host, const int32_t *parent, const void *q,
                                  const void *k_tree, const void *v_tree, const void *k_pages,
                                  const void *v_pages, int32_t num_pages, const int32_t *block_table,
                                  int32_t block_table_stride, const int32_t *prefix_len,
                                  const int32_t *prefix_len_host, int32_t num_q_heads, int32_t num_kv_heads,
                                  int32_t head_dim, int32_t page_size, float sm_scale, int32_t dtype,
                                  void *out, void *workspace, size_t workspace_bytes, void *stream) {
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
      make_plan(num_requests, node_indptr_host, prefix_len_host, num_kv_heads, shape.group, head_dim, dtype);
  if (plan.ws_bytes > 0) {
    if (!workspace || workspace_bytes < plan.ws_bytes)
      return fail(ADASERVE_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", plan.ws_bytes,
                  workspace ? workspace_bytes : (size_t)0);
    if (!aligned(workspace, 256)) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
  }
  st = check_device();
  if (st != ADASERVE_OK) return st;

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
  if (dtype == ADASERVE_BF16) fill_plan_table(a, num_requests, node_indptr_host, prefix_len_host, plan);
  a.sm_scale = sm_scale;
  a.scale_log2 = sm_scale * 1.4426950408889634f;
  hipStream_t s = (hipStream_t)stream;
  if (dtype == ADASERVE_BF16)
    return launch_status(launch_tree_attn_bf16(a, head_dim, plan.needs_combine, s), "tree attention launch");
  return launch_status(launch_tree_attn_f32(a, head_dim, s), "tree attention launch");
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
  return (size_t)total_nodes * 16;
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
  const size_t need = (size_t)total_nodes * 16;
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
  return launch_status(launch_sampled_accept(a, dtype == ADASERVE_BF16, (hipStream_t)stream), "sampled accept launch");
}

}  // extern "C"
