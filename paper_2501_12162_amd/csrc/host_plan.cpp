// Host-only part of the library (see host_plan.h): argument validation and
// the split-KV planner of the tree-attention entry points.
#include "host_plan.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <iterator>
#include <string>

namespace adaserve {

namespace {
thread_local std::string g_last_error;
}  // namespace

int32_t fail(int32_t code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

const char *last_error_message() { return g_last_error.c_str(); }

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

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
    if (L > kMaxPrefixLen) return fail(ADASERVE_ERR_UNSUPPORTED, "prefix_len[%d] = %d (max %d)", r, L, kMaxPrefixLen);
    if (bt_stride_or_neg >= 0 && ceil_div(L, kPageSize) > bt_stride_or_neg)
      return fail(ADASERVE_ERR_INVALID_ARGUMENT, "prefix_len[%d] = %d needs %d pages > block_table_stride %d", r, L,
                  ceil_div(L, kPageSize), bt_stride_or_neg);
  }
  if (total > INT32_MAX / 16) return fail(ADASERVE_ERR_INVALID_ARGUMENT, "too many tree nodes (%lld)", (long long)total);
  shape.total_nodes = (int32_t)total;
  return ADASERVE_OK;
}



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
  auto insert = [&runs](double load, int64_t slots) {
    auto it = std::lower_bound(runs.begin(), runs.end(), load,
                               [](const std::pair<double, int64_t> &x, double v) { return x.first < v; });
    if (it != runs.end() && it->first == load)
      it->second += slots;
    else
      runs.insert(it, {load, slots});
  };
  for (const auto &u : units) {
    const double t = u.first;
    int64_t c = u.second;
    // Units of duration t go one by one to a least-loaded slot.  The k0
    // slots of the lowest run take them in rounds, one per slot, until they
    // pass the next run's load (or the units run out): whole rounds move the
    // run up together; a last partial round splits it.
    while (c > 0) {
      const double x0 = runs.front().first;
      const int64_t k0 = runs.front().second;
      if (c < k0) {
        runs.front().second -= c;
        insert(x0 + t, c);
        break;
      }
      runs.erase(runs.begin());
      int64_t rounds = c / k0;
      if (!runs.empty())
        rounds = std::min<int64_t>(rounds, std::max<int64_t>(1, (int64_t)std::ceil((runs.front().first - x0) / t)));
      c -= rounds * k0;
      insert(x0 + (double)rounds * t, k0);
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
static AttnPlan evaluate_plan(int32_t B, const int32_t *indptr_host, const int32_t *plen_host, int32_t hkv,
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
  best.single_tile = true;
  for (int32_t r = 0; r < B; ++r)
    best.single_tile &= row_tiles(indptr_host[r + 1] - indptr_host[r], group, rt) == 1;
  return best;
}

AttnPlan make_plan_cached(int32_t B, const int32_t *indptr_host, const int32_t *plen_host, int32_t hkv,
                          int32_t group, int32_t head_dim, int32_t dtype) {
  if (dtype != ADASERVE_BF16 || B <= 0) return make_plan(B, indptr_host, plen_host, hkv, group, head_dim, dtype);
  struct Entry {
    bool valid = false;
    int32_t B = 0, hkv = 0, group = 0, head_dim = 0, dtype = 0;
    std::vector<int32_t> indptr, plen;
    AttnPlan plan;
  };
  thread_local Entry e;
  const bool hit = e.valid && e.B == B && e.hkv == hkv && e.group == group && e.head_dim == head_dim &&
                   e.dtype == dtype && std::equal(indptr_host, indptr_host + B + 1, e.indptr.begin()) &&
                   std::equal(plen_host, plen_host + B, e.plen.begin());
  if (!hit) {
    e.valid = false;
    e.plan = make_plan(B, indptr_host, plen_host, hkv, group, head_dim, dtype);
    e.indptr.assign(indptr_host, indptr_host + B + 1);
    e.plen.assign(plen_host, plen_host + B);
    e.B = B;
    e.hkv = hkv;
    e.group = group;
    e.head_dim = head_dim;
    e.dtype = dtype;
    e.valid = true;
  }
  return e.plan;
}

// Fills the dispatch-ordered request table (descending per-unit cost) when
// the batch fits in the kernel arguments; otherwise leaves it empty.
void fill_plan_table(PlanTable &t, int32_t B, const int32_t *indptr_host, const int32_t *plen_host,
                     int32_t num_kv_heads, int32_t group, const AttnPlan &p) {
  t.count = 0;
  t.merge_blocks = 0;
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
    end += (int64_t)num_kv_heads * row_tiles(n, group, p.rows_per_tile) *
           prefix_chunks(plen_host[r], p.chunk_len[r]);
    // merge blocks: 16 rows of one kv-head each, for split requests only
    if (prefix_chunks(plen_host[r], p.chunk_len[r]) > 1) gend += (int64_t)num_kv_heads * ceil_div(n * group, 16);
    t.entry[i].unit_end = (int32_t)end;
    t.entry[i].group_end = (int32_t)gend;
    t.entry[i].request_and_chunk = pack_request_chunk(r, p.chunk_len[r] / kKeysPerBlock);
    t.entry[i].node_base = indptr_host[r];
    t.entry[i].n_and_len = pack_nodes_len(n, plen_host[r]);
  }
  t.count = B;
  t.merge_blocks = gend;
}


}  // namespace adaserve
