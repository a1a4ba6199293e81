// Checks of the library's host-only code (argument validation, split-KV
// planner, plan-table packing), built with -fsanitize=address,undefined by
// tests/test_sanitizers.py.  Exits 1 on the first broken invariant; the
// sanitizers abort on any memory error or undefined behaviour.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <queue>
#include <random>
#include <set>
#include <vector>

#include "host_plan.h"

using namespace adaserve;

static int g_checks = 0;
#define CHECK(cond, ...)                                              \
  do {                                                                \
    ++g_checks;                                                       \
    if (!(cond)) {                                                    \
      std::fprintf(stderr, "FAILED %s:%d: %s: ", __FILE__, __LINE__, #cond); \
      std::fprintf(stderr, __VA_ARGS__);                              \
      std::fprintf(stderr, "\n");                                     \
      std::exit(1);                                                   \
    }                                                                 \
  } while (0)

struct Batch {
  std::vector<int32_t> indptr, plen;
};

static Batch random_batch(std::mt19937_64 &rng, int B, int max_nodes, int max_len) {
  Batch b;
  b.indptr.push_back(0);
  for (int r = 0; r < B; ++r) {
    const int n = 1 + (int)(rng() % (uint64_t)max_nodes);
    b.indptr.push_back(b.indptr.back() + n);
    int L;
    switch (rng() % 6) {
      case 0: L = 0; break;
      case 1: L = (int)(rng() % 64); break;
      case 2: L = 32 * (int)(rng() % 300) + (int)(rng() % 3) - 1; break;
      default: L = (int)(rng() % (uint64_t)(max_len + 1)); break;
    }
    b.plen.push_back(L < 0 ? 0 : L);
  }
  return b;
}

// Brute-force longest-first dealing onto kSlots equal slots (the planner's
// makespan model) with a heap.
static double brute_makespan(std::vector<std::pair<double, int64_t>> units, int slots) {
  std::vector<double> d;
  for (auto &u : units)
    for (int64_t i = 0; i < u.second; ++i) d.push_back(u.first);
  std::sort(d.begin(), d.end(), [](double x, double y) { return x > y; });
  std::priority_queue<double, std::vector<double>, std::greater<double>> q;
  for (int i = 0; i < slots; ++i) q.push(0.0);
  double mk = 0;
  for (double t : d) {
    double s = q.top();
    q.pop();
    s += t;
    mk = std::max(mk, s);
    q.push(s);
  }
  return mk;
}

static void check_plan(const Batch &b, int hq, int hkv, int D) {
  const int B = (int)b.plen.size();
  AttnShape shape;
  const int32_t st = validate_attn_shape(B, b.indptr.data(), b.plen.data(), hq, hkv, D, 16, ADASERVE_BF16, -1, shape);
  if (st != ADASERVE_OK) return;
  const int G = hq / hkv;
  const AttnPlan p = make_plan(B, b.indptr.data(), b.plen.data(), hkv, G, D, ADASERVE_BF16);
  CHECK((int)p.chunk_len.size() == B, "%zu chunk lengths for %d requests", p.chunk_len.size(), B);
  int64_t units = 0, groups = 0;
  bool split = false;
  for (int r = 0; r < B; ++r) {
    const int n = b.indptr[r + 1] - b.indptr[r];
    const int ck = p.chunk_len[r];
    CHECK(ck > 0 && ck <= kMaxChunk && ck % kKeysPerBlock == 0, "request %d chunk %d", r, ck);
    const int chunks = prefix_chunks(b.plen[r], ck);
    units += (int64_t)hkv * row_tiles(n, G, p.rows_per_tile) * chunks;
    groups += (int64_t)hkv * row_tiles(n, G, p.rows_per_tile);
    split |= chunks > 1;
    if (B > kPlanMax)  // without a plan table the device rebuilds the chunk lengths
      CHECK(ck == chunk_keys(n, G, p.rows_per_tile, p.chunk_target, p.chunk_floor), "request %d", r);
  }
  CHECK(units == p.units, "units %lld vs %lld", (long long)units, (long long)p.units);
  CHECK(groups == p.row_groups, "row groups");
  CHECK(split == p.needs_combine, "combine flag");
  bool one_tile = true;
  for (int r = 0; r < B; ++r) one_tile &= row_tiles(b.indptr[r + 1] - b.indptr[r], G, p.rows_per_tile) == 1;
  CHECK(one_tile == p.single_tile, "single-tile flag");
  CHECK((p.ws_bytes == 0) == !split, "workspace %zu", p.ws_bytes);
  if (split) {
    CHECK(p.ws_o_bytes >= (size_t)p.units * kMaxRowsPerTile * D * 2, "partial outputs");
    CHECK(p.ws_ml_bytes >= (size_t)p.units * kMaxRowsPerTile * 8, "partial max / sums");
    CHECK(p.ws_bytes == p.ws_o_bytes + p.ws_ml_bytes && p.ws_o_bytes % 256 == 0, "workspace layout");
  }
  CHECK(std::isfinite(p.est_us) && p.est_us > 0, "estimate %g", p.est_us);
  CHECK(p.padded_grid >= p.units && p.padded_grid % (kXcds * kXcdRun) == 0, "grid");
  if (p.padded_grid <= 4096) {
    std::vector<char> seen((size_t)p.padded_grid, 0);
    for (int64_t blk = 0; blk < p.padded_grid; ++blk) {
      const int64_t u = xcd_swizzle(blk, p.padded_grid);
      CHECK(u >= 0 && u < p.padded_grid && !seen[(size_t)u], "swizzle of %lld", (long long)blk);
      seen[(size_t)u] = 1;
    }
  }
  PlanTable t;
  fill_plan_table(t, B, b.indptr.data(), b.plen.data(), hkv, G, p);
  if (B > kPlanMax) {
    CHECK(t.count == 0, "table for %d requests", B);
    return;
  }
  CHECK(t.count == B, "table count");
  std::set<int> reqs;
  int64_t prev_end = 0, prev_g = 0, prev_cost = INT64_MAX;
  for (int i = 0; i < B; ++i) {
    const PlanEntry &e = t.entry[i];
    const int r = plan_request(e.request_and_chunk);
    CHECK(r >= 0 && r < B && reqs.insert(r).second, "entry %d request %d", i, r);
    const int n = b.indptr[r + 1] - b.indptr[r];
    CHECK(plan_nodes(e.n_and_len) == n, "nodes of %d", r);
    CHECK(plan_prefix_len(e.n_and_len) == b.plen[r], "prefix of %d", r);
    CHECK(plan_chunk_keys(e.request_and_chunk) == p.chunk_len[r], "chunk of %d", r);
    CHECK(e.node_base == b.indptr[r], "node base of %d", r);
    const int chunks = prefix_chunks(b.plen[r], p.chunk_len[r]);
    CHECK(e.unit_end - prev_end == (int64_t)hkv * row_tiles(n, G, p.rows_per_tile) * chunks, "units of %d", r);
    CHECK(e.group_end - prev_g == (chunks > 1 ? (int64_t)hkv * ceil_div(n * G, 16) : 0), "merge blocks of %d", r);
    const int64_t cost = std::min(b.plen[r], p.chunk_len[r]) + n;
    CHECK(cost <= prev_cost, "dispatch order at %d", i);
    prev_end = e.unit_end;
    prev_g = e.group_end;
    prev_cost = cost;
  }
  CHECK(prev_end == p.units && prev_g == t.merge_blocks, "table totals");
}

static bool same_plan(const AttnPlan &x, const AttnPlan &y) {
  return x.rows_per_tile == y.rows_per_tile && x.chunk_target == y.chunk_target && x.chunk_floor == y.chunk_floor &&
         x.chunk_len == y.chunk_len && x.units == y.units && x.padded_grid == y.padded_grid &&
         x.row_groups == y.row_groups && x.needs_combine == y.needs_combine && x.single_tile == y.single_tile &&
         x.ws_o_bytes == y.ws_o_bytes &&
         x.ws_ml_bytes == y.ws_ml_bytes && x.ws_bytes == y.ws_bytes && x.est_us == y.est_us;
}

// The cached planner against a fresh plan on every call of a sequence that
// repeats batches, refills the same buffers in place (one prefix grows by a
// token, one tree loses a node) and changes only a scalar argument.
static void check_plan_cache(std::mt19937_64 &rng) {
  std::vector<int32_t> ip, pl;
  for (int it = 0; it < 400; ++it) {
    const int op = (int)(rng() % 5);
    if (ip.empty() || op == 0) {
      const Batch b = random_batch(rng, 1 + (int)(rng() % 40), 64, 20000);
      ip = b.indptr;
      pl = b.plen;
    } else if (op == 1) {
      pl[rng() % pl.size()] += 1;
    } else if (op == 2) {
      const size_t r = rng() % pl.size();
      if (ip[r + 1] - ip[r] > 1)
        for (size_t i = r + 1; i < ip.size(); ++i) ip[i] -= 1;
    }  // op 3, 4: the same contents again
    const int B = (int)pl.size();
    const int hkv = op == 4 ? 2 : 8, G = op == 4 ? 16 : 4, D = it % 2 ? 128 : 64;
    const AttnPlan fresh = make_plan(B, ip.data(), pl.data(), hkv, G, D, ADASERVE_BF16);
    const AttnPlan cached = make_plan_cached(B, ip.data(), pl.data(), hkv, G, D, ADASERVE_BF16);
    CHECK(same_plan(fresh, cached), "cached plan differs at step %d (op %d)", it, op);
    CHECK(same_plan(fresh, make_plan_cached(B, ip.data(), pl.data(), hkv, G, D, ADASERVE_BF16)),
          "second cached call differs at step %d", it);
  }
  CHECK(make_plan_cached(0, nullptr, nullptr, 8, 4, 128, ADASERVE_BF16).units == 0, "empty batch");
}

int main() {
  std::mt19937_64 rng(2501);
  // validation: malformed host mirrors and scalars give a status, never UB
  for (int it = 0; it < 20000; ++it) {
    const int B = (int)(rng() % 8);
    std::vector<int32_t> ip(B + 1), pl(B);
    for (auto &x : ip) x = (int32_t)(rng() % 3 == 0 ? rng() : rng() % 300) - (rng() % 7 == 0 ? 200 : 0);
    for (auto &x : pl) x = (int32_t)(rng() % 4 == 0 ? rng() : rng() % 40000) - (rng() % 9 == 0 ? 5 : 0);
    const int hq = (int)(rng() % 70) - 2, hkv = (int)(rng() % 20) - 2, D = rng() % 3 ? 128 : (int)(rng() % 300);
    AttnShape shape;
    const int32_t st = validate_attn_shape(B, ip.data(), pl.data(), hq, hkv, D, rng() % 5 ? 16 : 8,
                                           (int)(rng() % 3), (int)(rng() % 3000) - 1, shape);
    CHECK(st >= ADASERVE_OK && st <= ADASERVE_ERR_DEVICE, "status %d", st);
    CHECK(st != ADASERVE_OK || shape.total_nodes >= B, "accepted a batch with %d nodes", shape.total_nodes);
    if (st != ADASERVE_OK) CHECK(last_error_message()[0] != 0, "no message");
  }
  // planner on valid batches: small, named-workload-like and extreme shapes
  const int heads[][2] = {{32, 8}, {64, 8}, {8, 2}, {16, 16}, {32, 2}, {4, 2}, {16, 1}};
  for (int it = 0; it < 600; ++it) {
    const auto &h = heads[it % 7];
    const int B = 1 + (int)(rng() % (it % 5 == 0 ? 300 : 64));
    const Batch b = random_batch(rng, B, it % 3 ? 128 : 8, it % 4 ? 20000 : 200000);
    check_plan(b, h[0], h[1], it % 2 ? 128 : 64);
  }
  {
    Batch b;  // the longest prefixes the validation accepts, the largest trees
    b.indptr = {0, 128, 256};
    b.plen = {kMaxPrefixLen, kMaxPrefixLen - 31};
    check_plan(b, 32, 2, 128);
    check_plan(b, 128, 8, 64);
  }
  {
    Batch b;  // exactly kPlanMax requests and one more
    for (int extra = 0; extra < 2; ++extra) {
      b.indptr = {0};
      b.plen.clear();
      for (int r = 0; r < kPlanMax + extra; ++r) {
        b.indptr.push_back(b.indptr.back() + 1 + r % 128);
        b.plen.push_back(r * 97);
      }
      check_plan(b, 32, 8, 128);
    }
  }
  check_plan_cache(rng);
  // the makespan model against brute-force dealing
  for (int it = 0; it < 300; ++it) {
    std::vector<std::pair<double, int64_t>> u;
    const int k = 1 + (int)(rng() % 6);
    for (int i = 0; i < k; ++i) u.push_back({1.0 + (double)(rng() % 40), 1 + (int64_t)(rng() % 700)});
    auto copy = u;
    const double fast = lpt_makespan(copy);
    const double slow = brute_makespan(u, 512);
    CHECK(std::fabs(fast - slow) < 1e-9, "makespan %g vs %g", fast, slow);
  }
  std::printf("host plan checks passed: %d\n", g_checks);
  return 0;
}
