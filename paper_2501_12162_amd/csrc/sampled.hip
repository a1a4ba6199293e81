// Tree verification for sampled decoding on gfx950: multi-step speculative
// sampling over each request's draft token tree (the tree-based verification
// of prior work that section 4.3 step 4 delegates to).
//
// From the root, the children of the current node u are tried in index
// order; child c with token t is accepted when u_accept[c] * q_u(t) <
// p_res(t), p_u / q_u being the target / draft softmax at u and p_res
// starting as p_u; a rejection replaces p_res by max(0, p_res - q_u),
// renormalised.  An accepted child becomes the current node; otherwise the
// bonus token is drawn from p_res (inverse CDF at u_bonus[u]) and the walk
// ends.
//
// Every residual has the closed form max(0, p - c q) / S: after a
// rejection c grows by the previous S and S is the new residual's mass
// (if p_res = r/S with r = max(0, p - c q), then max(0, p_res - q) is
// proportional to max(0, p - (c + S) q)).  A first kernel computes every
// node's softmax statistics (max and exp-sum of its target row, and of its
// draft row when it has children) across the whole chip, in parts that
// follow the token ranges ("rounds", at most 64) of the draw below; the
// walk -- one workgroup of 1024 threads per request -- then reads them, so
// an acceptance test costs two logits, a rejection one pass over the node's
// two rows (the new S; none after the node's last child, whose residual the
// draw sums anyway), and the bonus draw the residual's mass in each round
// (from the statistics parts for p itself, else one pass over both rows),
// then a pass over the one round that holds its target.  The acceptance
// tests' inputs depend on the tree alone, so the walk
// loads them all, a thread per node, before it starts; the same holds for
// each node's first test (p_res is still p_u), which those threads also
// take, so a run of accepted first children costs one LDS read per node.
#include <type_traits>

#include "device_common.h"
#include "kernels.h"

namespace adaserve {

namespace {

constexpr int kThreads = 1024;
constexpr int kStatsThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kGroupVecs = kSampledGroupVecs;  // 16-byte vectors per pass iteration (four per thread)
constexpr int kMaxRounds = kSampledMaxRounds;  // token ranges whose masses a pass keeps (one per lane)
static_assert(kGroupVecs == 4 * kThreads, "a group is four vectors per thread");

template <bool BF16>
__device__ __forceinline__ float elem(const u32x4 &w, int e) {
  if (BF16) return __uint_as_float((e & 1) ? (w[e >> 1] & 0xffff0000u) : (w[e >> 1] << 16));
  return __uint_as_float(w[e]);
}

template <bool BF16>
__device__ __forceinline__ float load_one(const void *row, int v) {
  if (BF16) return bf16_bits_to_float(((const uint16_t *)row)[v]);
  return ((const float *)row)[v];
}

struct Shared {
  int32_t parent[kMaxSampledNodes];
  int32_t token[kMaxSampledNodes];
  int32_t path[kMaxSampledNodes];
  int32_t out[kMaxSampledNodes];
  uint32_t kids[kMaxSampledNodes][kMaxSampledNodes / 32];  // bit c: node c is a child
  // for each node c: the two logits of c's token at its parent, c's
  // acceptance uniform and c's own softmax statistics (the root: only its
  // statistics)
  float kid_p[kMaxSampledNodes];
  float kid_q[kMaxSampledNodes];
  float kid_u[kMaxSampledNodes];
  float4 kid_st[kMaxSampledNodes];
  int32_t fwd[kMaxSampledNodes];  // node's first child when it passes its test, else -1
  float red_a[kWaves];
  float scan[kWaves];  // the draw's per-wave sums
  float rsum[kMaxRounds][kWaves];  // per round and wave: the residual's mass
  float cum[kMaxRounds];           // inclusive prefix of the rounds' masses, in token order
  int32_t bad;
  int32_t pick;
};

// Block-wide sum (every thread gets it).
__device__ float block_sum(float v, Shared &sh) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) sh.red_a[wave] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) t += sh.red_a[w];
  __syncthreads();
  return t;
}

// A residual max(0, p(v) - c q(v)) (p itself when c = 0 or the node has no
// child, hence no q), p = exp(x - mp) * ip and q = exp(y - mq) * iq.
struct Residual {
  float mp, ip, mq, iq, c;
  bool has_q;
};

// Its unnormalised mass at token v, as the passes over a row evaluate it.
// The normalisers and c go into the exponents, p = 2^(x log2 e + op) and
// c q = 2^(y log2 e + oq), so a logit costs one FMA and one exp2 (a pass is
// bound by one CU's ALU; the offsets are rounded once per pass, ~1e-6
// relative to the terms).  Whether q enters (Q: the node has a child and
// c != 0) is a template argument of the passes, so their loads are straight
// -line code (a load under a branch makes the compiler wait for it before
// the next).  (Bulk sums use the hardware exp2, which flushes results below
// 2^-126 to zero: such terms are far below the sums' rounding.)
template <bool Q>
struct ResidualPass {
  static constexpr bool kQ = Q;
  float op, oq;
  __device__ explicit ResidualPass(const Residual &R)
      : op(-R.mp * kLog2e + log2f(R.ip)), oq(Q ? -R.mq * kLog2e + log2f(R.c * R.iq) : 0.f) {}
  __device__ __forceinline__ float at(float x, float y) const {
    const float p = __builtin_amdgcn_exp2f(fmaf(x, kLog2e, op));
    if constexpr (!Q) return p;
    return fmaxf(p - __builtin_amdgcn_exp2f(fmaf(y, kLog2e, oq)), 0.f);
  }
};

__device__ __forceinline__ bool q_enters(const Residual &R) { return R.has_q && R.c != 0.f; }

// Round layout of a pass over a row: its 16-byte vectors go in groups of
// kGroupVecs (in a group, thread t takes vectors t, t + kThreads, t +
// 2 kThreads and t + 3 kThreads, so the loads coalesce); gpr consecutive
// groups form a round, a contiguous token range, at most kMaxRounds of them.
// The tokens past the last whole vector belong to the last round.  The
// statistics pass keeps its parts inside these rounds.
using Rounds = SampledRounds;

// Sum over the vocabulary of the residual.
template <bool BF16, class RT>
__device__ float residual_mass_t(const char *prow, const char *qrow, int vocab, const RT &R, Shared &sh) {
  constexpr int EPV = BF16 ? 8 : 4;
  const int nvec = vocab / EPV;
  float s = 0.f;
  int i = threadIdx.x;
  // four vectors of each row in flight per thread
  for (; i + 3 * kThreads < nvec; i += 4 * kThreads) {
    u32x4 w[4], z[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      w[k] = *(const u32x4 *)(prow + (int64_t)(i + k * kThreads) * 16);
      z[k] = RT::kQ ? *(const u32x4 *)(qrow + (int64_t)(i + k * kThreads) * 16) : w[k];
    }
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int e = 0; e < EPV; ++e) s += R.at(elem<BF16>(w[k], e), elem<BF16>(z[k], e));
  }
  for (; i < nvec; i += kThreads) {
    const u32x4 w = *(const u32x4 *)(prow + (int64_t)i * 16);
    const u32x4 z = RT::kQ ? *(const u32x4 *)(qrow + (int64_t)i * 16) : w;
#pragma unroll
    for (int e = 0; e < EPV; ++e) s += R.at(elem<BF16>(w, e), elem<BF16>(z, e));
  }
  for (int v = nvec * EPV + threadIdx.x; v < vocab; v += kThreads)
    s += R.at(load_one<BF16>(prow, v), RT::kQ ? load_one<BF16>(qrow, v) : 0.f);
  return block_sum(s, sh);
}

template <bool BF16>
__device__ float residual_mass(const char *prow, const char *qrow, int vocab, const Residual &R, Shared &sh) {
  if (q_enters(R)) return residual_mass_t<BF16>(prow, qrow, vocab, ResidualPass<true>(R), sh);
  return residual_mass_t<BF16>(prow, qrow, vocab, ResidualPass<false>(R), sh);
}

// The residual's mass in each round (per wave in sh.rsum, then the
// inclusive prefix over the rounds in sh.cum), for the bonus draw; returns
// the total, the last prefix, so the two always agree.  (A rejection needs
// only the total: residual_mass above, whose loop measured faster.)
template <bool BF16, class RT>
__device__ float residual_rounds(const char *prow, const char *qrow, int vocab, const RT &R, Shared &sh) {
  constexpr int EPV = BF16 ? 8 : 4;
  const Rounds rd(vocab, EPV);
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  float acc = 0.f;
  // round r's mass, summed over the wave, goes to sh.rsum[r][wave]
  auto flush = [&](int g) {
    const float ws = wave_sum(acc);
    if (lane == 0) sh.rsum[g / rd.gpr][wave] = ws;
    acc = 0.f;
  };
  const int nfull = rd.nvec / kGroupVecs;  // groups whose four vectors every thread has
  for (int g = 0; g < nfull; ++g) {
    // four vectors of each row in flight per thread
    const int i0 = g * kGroupVecs + t;
    u32x4 w[4], z[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      w[k] = *(const u32x4 *)(prow + (int64_t)(i0 + k * kThreads) * 16);
      z[k] = RT::kQ ? *(const u32x4 *)(qrow + (int64_t)(i0 + k * kThreads) * 16) : w[k];
    }
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int e = 0; e < EPV; ++e) acc += R.at(elem<BF16>(w[k], e), elem<BF16>(z[k], e));
    if ((g + 1) % rd.gpr == 0 && g + 1 < rd.ngroups) flush(g);
  }
  // the last, partial group (when there is one) and the tokens past the last vector
  for (int i = nfull * kGroupVecs + t; i < rd.nvec; i += kThreads) {
    const u32x4 w = *(const u32x4 *)(prow + (int64_t)i * 16);
    const u32x4 z = RT::kQ ? *(const u32x4 *)(qrow + (int64_t)i * 16) : w;
#pragma unroll
    for (int e = 0; e < EPV; ++e) acc += R.at(elem<BF16>(w, e), elem<BF16>(z, e));
  }
  for (int v = rd.nvec * EPV + t; v < vocab; v += kThreads)
    acc += R.at(load_one<BF16>(prow, v), RT::kQ ? load_one<BF16>(qrow, v) : 0.f);
  flush(rd.ngroups - 1);
  __syncthreads();
  if (wave == 0) {
    // lane k: round k's mass, then the inclusive prefix over the rounds
    float m = 0.f;
    if (lane < rd.nrounds)
      for (int w = 0; w < kWaves; ++w) m += sh.rsum[lane][w];
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float o = __shfl_up(m, off, 64);
      if (lane >= off) m += o;
    }
    if (lane < rd.nrounds) sh.cum[lane] = m;
  }
  __syncthreads();
  return sh.cum[rd.nrounds - 1];
}

// Inverse-CDF draw from the residual: the smallest v whose cumulative mass
// (in token order) exceeds u * (total mass); the last token of nonzero mass
// when rounding leaves the target past the end (-1 when no token has mass).
// With the rounds' masses in sh.cum (inclusive prefix), the round that holds
// the target is read, each thread taking a contiguous run of its vectors so
// that per-thread sums scan in token order.
template <bool BF16, class RT>
__device__ int draw_in_rounds(const char *prow, const char *qrow, int vocab, const RT &R, float u, Shared &sh) {
  constexpr int EPV = BF16 ? 8 : 4;
  const Rounds rd(vocab, EPV);
  const int t = threadIdx.x, lane = t & 63;
  const float total = sh.cum[rd.nrounds - 1];
  const float target = u * total;
  // the first round whose prefix exceeds the target, else the last round
  // with mass (its last token of nonzero mass is the answer)
  const bool in = lane < rd.nrounds;
  const float cl = in ? sh.cum[lane] : 0.f;
  const float cp = in && lane > 0 ? sh.cum[lane - 1] : 0.f;
  const uint64_t over = __ballot(in && cl > target);
  const uint64_t grows = __ballot(in && cl > cp);
  if (!grows) return -1;
  const bool find = over != 0;
  const int rs = find ? __ffsll((unsigned long long)over) - 1 : 63 - __clzll((unsigned long long)grows);
  const float before = rs > 0 ? sh.cum[rs - 1] : 0.f;

  const int64_t vb = (int64_t)rs * rd.gpr * kGroupVecs;
  const int64_t ve = min((int64_t)rd.nvec, vb + (int64_t)rd.gpr * kGroupVecs);
  const int cv = 4 * rd.gpr;  // vectors per thread
  const int64_t tv0 = min(ve, vb + (int64_t)t * cv), tv1 = min(ve, tv0 + cv);
  const bool tail = rs == rd.nrounds - 1 && t == kThreads - 1;  // tokens past the last vector
  // one pass over this thread's tokens, in order: their mass, the last one
  // with mass, and (find) the first at which start + running mass > goal.
  // The vectors go through w / z four at a time; when the run is one such
  // chunk (always for rounds of one group) of the target row alone, a second
  // pass reuses them (both rows' would not fit the registers).
  u32x4 w[4], z[4];
  const bool one_chunk = !RT::kQ && tv1 - tv0 <= 4;
  auto run = [&](float start, float goal, bool stop, bool reuse, int &found, int &last) {
    float acc = start;
    found = -1;
    last = -1;
    for (int64_t i = tv0; i < tv1; i += 4) {
      if (!reuse) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int64_t j = min(i + k, tv1 - 1);
          w[k] = *(const u32x4 *)(prow + j * 16);
          z[k] = RT::kQ ? *(const u32x4 *)(qrow + j * 16) : w[k];
        }
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        // a slot past the run (its load repeats the run's last vector) adds
        // exactly nothing and moves neither `last` nor `found`; masking it
        // rather than leaving the loop keeps the loads above straight-line
        const bool in_run = i + k < tv1;
#pragma unroll
        for (int e = 0; e < EPV; ++e) {
          const float r = in_run ? R.at(elem<BF16>(w[k], e), elem<BF16>(z[k], e)) : 0.f;
          acc += r;
          const int v = (int)((i + k) * EPV) + e;
          if (r > 0.f) last = v;
          if (stop && found < 0 && acc > goal) found = v;
        }
      }
    }
    if (tail)
      for (int v = rd.nvec * EPV; v < vocab; ++v) {
        const float r = R.at(load_one<BF16>(prow, v), RT::kQ ? load_one<BF16>(qrow, v) : 0.f);
        acc += r;
        if (r > 0.f) last = v;
        if (stop && found < 0 && acc > goal) found = v;
      }
    return acc - start;
  };
  int found, last;
  const float s = run(0.f, 0.f, false, false, found, last);
  // inclusive prefix of the threads' sums within the round: by shuffles
  // within each wave, then each wave's offset as the sequential sum of the
  // earlier waves' totals, so that every thread's start is bit for bit the
  // previous thread's end (exactly one thread holds the target)
  float x = s;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const float o = __shfl_up(x, off, 64);
    if (lane >= off) x += o;
  }
  const int wave = t >> 6;
  if (lane == 63) sh.scan[wave] = x;
  if (t == 0) sh.pick = -1;
  __syncthreads();
  float woff = 0.f;
  for (int k = 0; k < wave; ++k) woff += sh.scan[k];
  const float xprev = __shfl_up(x, 1, 64);
  const float lo = before + (lane > 0 ? woff + xprev : woff);
  const float hi = before + (woff + x);
  if (find && s > 0.f && lo <= target && target < hi) {
    int f, l2;
    run(lo, target, true, one_chunk, f, l2);
    sh.pick = f >= 0 ? min(f, last) : last;
  }
  __syncthreads();
  int pick = sh.pick;
  if (pick < 0) {
    // the round's last token of nonzero mass
    int lastv = last;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) lastv = max(lastv, __shfl_xor(lastv, off, 64));
    if ((t & 63) == 0) sh.red_a[t >> 6] = __int_as_float(lastv);
    __syncthreads();
    pick = -1;
    for (int w = 0; w < kWaves; ++w) pick = max(pick, __float_as_int(sh.red_a[w]));
    __syncthreads();
  }
  return pick;
}

// The rounds' masses of the target distribution p itself (nothing rejected
// at the node), from the statistics pass's parts of the node's row: `sub`
// consecutive parts per round, part j's (max, sum) rescaled to the node's
// (R.mp, 1 / R.ip); inclusive prefix into sh.cum.  No pass over the row.
__device__ void target_rounds(const Residual &R, const float4 *parts, int sub, int nrounds, Shared &sh) {
  const int t = threadIdx.x;
  if (t < 64) {
    float m = 0.f;
    if (t < nrounds * sub) {
      const float4 e = parts[t];
      if (e.x > -INFINITY) m = e.y * exp2f((e.x - R.mp) * kLog2e) * R.ip;
    }
    float rm = 0.f;  // lane r: round r's mass (nrounds * sub <= 64 lanes)
    for (int k = 0; k < sub; ++k) rm += __shfl(m, min(t * sub + k, 63), 64);
    if (t >= nrounds) rm = 0.f;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float o = __shfl_up(rm, off, 64);
      if (t >= off) rm += o;
    }
    if (t < nrounds) sh.cum[t] = rm;
  }
  __syncthreads();
}

// The bonus draw: from p itself, the rounds' masses come from the statistics
// parts (one read of one round); with q in the residual, one coalesced pass
// over both rows sums them first.
template <bool BF16>
__device__ int residual_draw(const char *prow, const char *qrow, int vocab, const Residual &R, float u,
                             const float4 *parts, int sub, Shared &sh) {
  if (q_enters(R)) {
    const ResidualPass<true> P(R);
    residual_rounds<BF16>(prow, qrow, vocab, P, sh);
    return draw_in_rounds<BF16>(prow, qrow, vocab, P, u, sh);
  }
  target_rounds(R, parts, sub, Rounds(vocab, BF16 ? 8 : 4).nrounds, sh);
  return draw_in_rounds<BF16>(prow, qrow, vocab, ResidualPass<false>(R), u, sh);
}

// Whether node g may have a child, so that its draft row is needed (q_g
// enters only the tests of g's children and the residuals at g).  The
// request that holds g is found by a 64-ary search of node_indptr (ballots
// over one wave's loads), then its later nodes are checked for g's local id
// as their parent.  Whatever does not fit a well-formed batch (node_indptr
// not increasing, a request longer than kMaxSampledNodes) answers true, so
// the row is read.  Wave-uniform.
__device__ bool node_may_have_children(const SampledArgs &a, int g) {
  const int lane = threadIdx.x & 63;
  int lo = 0, hi = a.num_requests;  // the request is in [lo, hi)
  while (hi - lo > 1) {
    const int step = (hi - lo + 63) / 64;
    const int k = lo + lane * step;
    const uint64_t m = __ballot(k < hi && a.node_indptr[k] <= g);
    if (!m) return true;
    lo += (63 - __clzll((unsigned long long)m)) * step;
    hi = min(hi, lo + step);
  }
  const int base = a.node_indptr[lo], end = a.node_indptr[lo + 1];
  if (!(base <= g && g < end && end - base <= kMaxSampledNodes && end <= a.total_nodes)) return true;
  bool kid = false;
  for (int j = g + 1 + lane; j < end; j += 64) kid |= a.parent[j] == g - base;
  return __ballot(kid) != 0;
}

// Softmax statistics of every node's target and draft rows, both rows in one
// pass: stats_parts workgroups per node, stats_sub contiguous pieces of each
// round (the last also takes the tokens past the last vector);
// stats[node * stats_parts + part] = (max_p, sum_p, max_q, sum_q) of part
// `part`; a leaf's draft row is not read (max_q = -inf, sum_q = 0).  The walk merges them into the node's statistics, and a bonus draw
// from p reads its rounds' masses off them.  The rows are streamed with the
// non-temporal hint: the walks read only the few rows they visit again, and
// they find those no slower for it (every batch measured faster streamed).
template <bool BF16>
__global__ __launch_bounds__(kStatsThreads) void sampled_stats_kernel(SampledArgs a) {
  constexpr int EPV = BF16 ? 8 : 4;
  constexpr int ESZ = BF16 ? 2 : 4;
  __shared__ float red[4][kStatsThreads / 64];
  const int node = blockIdx.x / a.stats_parts, part = blockIdx.x % a.stats_parts;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const char *prow = (const char *)a.target_logits + (int64_t)node * a.row_stride * ESZ;
  const char *qrow = (const char *)a.draft_logits + (int64_t)node * a.row_stride * ESZ;
  float mp = -INFINITY, sp = 0.f, mq = -INFINITY, sq = 0.f;
  auto add = [](float &m, float &s, float x) {
    const float nm = fmaxf(m, x);
    if (nm > -INFINITY) {
      s = (m > -INFINITY ? s * exp2f((m - nm) * kLog2e) : 0.f) + exp2f((x - nm) * kLog2e);
      m = nm;
    }
  };
  const Rounds rd(a.vocab, EPV);
  const int nvec = rd.nvec;
  const int round = part / a.stats_sub, piece = part % a.stats_sub;
  const int64_t r0 = (int64_t)round * rd.gpr * kGroupVecs;
  const int64_t r1 = min((int64_t)nvec, r0 + (int64_t)rd.gpr * kGroupVecs);
  const int vb = (int)(r0 + (r1 - r0) * piece / a.stats_sub);
  const int ve = (int)(r0 + (r1 - r0) * (piece + 1) / a.stats_sub);
  auto load = [&](const char *row, int i) -> u32x4 {
    return __builtin_nontemporal_load((const u32x4 *)(row + (int64_t)i * 16));
  };
  // one vector of a row into its running (max, sum) pair
  auto take = [&](const u32x4 &w, float &m, float &s) {
    float wm = elem<BF16>(w, 0);
#pragma unroll
    for (int e = 1; e < EPV; ++e) wm = fmaxf(wm, elem<BF16>(w, e));
    const float nm = fmaxf(m, wm);
    if (nm > -INFINITY) {
      float acc = 0.f;
#pragma unroll
      for (int e = 0; e < EPV; ++e) acc += __builtin_amdgcn_exp2f((elem<BF16>(w, e) - nm) * kLog2e);
      s = (m > -INFINITY ? s * __builtin_amdgcn_exp2f((m - nm) * kLog2e) : 0.f) + acc;
      m = nm;
    }
  };
  // The pass over the target row, and the draft row when Q: four vectors of
  // each row in flight per thread, all loads written before the first use
  // (the branches of `take` end the scheduler's regions, so it cannot hoist
  // later loads above them; and with the draft row's loads under a runtime
  // test, the compiler would wait for them all at its join).
  // A part is a few vectors per thread (about 8 of each row at 128256
  // logits and 8 parts), so its last, partial batch is taken the same way:
  // slots past the part load its last vector again and are taken as -inf
  // vectors, which leave every sum bit unchanged (each row is still taken in
  // the same order).
  constexpr uint32_t kNegInf = BF16 ? 0xff80ff80u : 0xff800000u;
  const u32x4 neg_inf = {kNegInf, kNegInf, kNegInf, kNegInf};
  auto pass = [&](auto with_q) {
    constexpr bool Q = decltype(with_q)::value;
    for (int i = vb + t; i < ve; i += 4 * kStatsThreads) {
      u32x4 w[4], z[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int j = min(i + k * kStatsThreads, ve - 1);
        w[k] = load(prow, j);
        if constexpr (Q) z[k] = load(qrow, j);
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const bool in = i + k * kStatsThreads < ve;
        take(in ? w[k] : neg_inf, mp, sp);
        if constexpr (Q) take(in ? z[k] : neg_inf, mq, sq);
      }
    }
    for (int v = nvec * EPV + t; part == a.stats_parts - 1 && v < a.vocab; v += kStatsThreads) {
      add(mp, sp, load_one<BF16>(prow, v));
      if constexpr (Q) add(mq, sq, load_one<BF16>(qrow, v));
    }
  };
  if (node_may_have_children(a, node))
    pass(std::true_type{});
  else
    pass(std::false_type{});
  // (max, sum) pairs over the workgroup
  float wmp = mp, wmq = mq;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    wmp = fmaxf(wmp, __shfl_xor(wmp, o, 64));
    wmq = fmaxf(wmq, __shfl_xor(wmq, o, 64));
  }
  float wsp = wmp > -INFINITY && mp > -INFINITY ? sp * exp2f((mp - wmp) * kLog2e) : 0.f;
  float wsq = wmq > -INFINITY && mq > -INFINITY ? sq * exp2f((mq - wmq) * kLog2e) : 0.f;
  wsp = wave_sum(wsp);
  wsq = wave_sum(wsq);
  if (lane == 0) {
    red[0][wave] = wmp;
    red[1][wave] = wsp;
    red[2][wave] = wmq;
    red[3][wave] = wsq;
  }
  __syncthreads();
  if (t == 0) {
    float Mp = -INFINITY, Mq = -INFINITY, Sp = 0.f, Sq = 0.f;
    for (int w = 0; w < kStatsThreads / 64; ++w) {
      Mp = fmaxf(Mp, red[0][w]);
      Mq = fmaxf(Mq, red[2][w]);
    }
    for (int w = 0; w < kStatsThreads / 64; ++w) {
      if (red[0][w] > -INFINITY) Sp += red[1][w] * exp2f((red[0][w] - Mp) * kLog2e);
      if (red[2][w] > -INFINITY) Sq += red[3][w] * exp2f((red[2][w] - Mq) * kLog2e);
    }
    a.stats[blockIdx.x] = make_float4(Mp, Sp, Mq, Sq);
  }
}

template <bool BF16>
__global__ __launch_bounds__(kThreads) void sampled_accept_kernel(SampledArgs a) {
  __shared__ Shared sh;
  constexpr int ESZ = BF16 ? 2 : 4;
  const int r = blockIdx.x, t = threadIdx.x;
  const int K = a.max_accept;
  int32_t *alen = a.accept_len + r;
  int32_t *otok = a.accept_tokens + (int64_t)r * K;
  int32_t *onode = a.accept_nodes + (int64_t)r * K;

  const int32_t base = a.node_indptr[r];
  const int32_t n = a.node_indptr[r + 1] - base;
  const bool shape_ok = n >= 1 && n <= kMaxSampledNodes && base >= 0 && base + n <= a.total_nodes;
  if (t == 0) sh.bad = shape_ok ? 0 : 1;
  if (shape_ok) {
    // every node's children as a bit set, built below for the walk (which
    // takes a node's children in index order: lowest set bit first)
    uint32_t *words = &sh.kids[0][0];
    for (int i = t; i < n * (kMaxSampledNodes / 32); i += kThreads) words[i] = 0u;
  }
  __syncthreads();
  // A thread per node (n <= kMaxSampledNodes < kThreads): its parent and
  // token, checked; its uniform and statistics in the same round of loads;
  // then, for a well-formed node, its token's two logits at its parent.
  // Every test input depends on the tree alone, not on the path the walk
  // takes, so the walk reads global memory only in its passes.
  static_assert(kMaxSampledNodes <= kThreads, "a thread per node");
  if (shape_ok && t < n) {
    const int32_t p = a.parent[base + t];
    const int32_t tk = a.draft_tokens[base + t];
    const float ua = t > 0 ? a.u_accept[base + t] : 0.f;
    // the parts' (max, sum) pairs merged; one part is taken as it is
    const int np = a.stats_parts;
    const float4 *ps = a.stats + (int64_t)(base + t) * np;
    float4 st = ps[0];
    if (np > 1) {
      // eight parts' loads at a time, merged into running (max, sum) pairs
      float mp = -INFINITY, mq = -INFINITY, sp = 0.f, sq = 0.f;
      for (int j0 = 0; j0 < np; j0 += 8) {
        float4 pp[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) pp[k] = ps[min(j0 + k, np - 1)];
        float cp = mp, cq = mq;
#pragma unroll
        for (int k = 0; k < 8; ++k)
          if (j0 + k < np) {
            cp = fmaxf(cp, pp[k].x);
            cq = fmaxf(cq, pp[k].z);
          }
        sp = mp > -INFINITY ? sp * exp2f((mp - cp) * kLog2e) : 0.f;
        sq = mq > -INFINITY ? sq * exp2f((mq - cq) * kLog2e) : 0.f;
#pragma unroll
        for (int k = 0; k < 8; ++k)
          if (j0 + k < np) {
            if (pp[k].x > -INFINITY) sp += pp[k].y * exp2f((pp[k].x - cp) * kLog2e);
            if (pp[k].z > -INFINITY) sq += pp[k].w * exp2f((pp[k].z - cq) * kLog2e);
          }
        mp = cp;
        mq = cq;
      }
      st = make_float4(mp, sp, mq, sq);
    }
    sh.parent[t] = p;
    sh.token[t] = tk;
    sh.kid_st[t] = st;
    sh.kid_u[t] = ua;
    const bool ok = t == 0 ? p == -1 : (p >= 0 && p < t && tk >= 0 && tk < a.vocab);
    if (!ok) {
      atomicOr(&sh.bad, 1);
    } else if (t > 0) {
      atomicOr(&sh.kids[p][t >> 5], 1u << (t & 31));
      const int64_t prow_off = (int64_t)(base + p) * a.row_stride;
      sh.kid_p[t] = load_one<BF16>((const char *)a.target_logits + prow_off * ESZ, tk);
      sh.kid_q[t] = load_one<BF16>((const char *)a.draft_logits + prow_off * ESZ, tk);
    }
  }
  __syncthreads();
  if (!sh.bad) {
    // every node's depth must be below the output rows (K): each thread
    // follows its node's parent chain, at most K steps (parents come first,
    // checked above, so every chain reaches the root).  A node with children
    // needs its draft statistics: max_q = -inf means that its draft row has
    // no logit above -inf (q is no distribution), or that the statistics
    // pass took it for a leaf (a node_indptr that is not increasing); either
    // way the request is not verified.
    if (t < n) {
      int v = t, d = 0;
      while (v != 0 && d < K) {
        v = sh.parent[v];
        ++d;
      }
      const bool has_kids = (sh.kids[t][0] | sh.kids[t][1] | sh.kids[t][2] | sh.kids[t][3]) != 0u;
      if (d >= K || (has_kids && !(sh.kid_st[t].z > -INFINITY))) atomicOr(&sh.bad, 1);
    }
  }
  __syncthreads();
  if (sh.bad) {
    for (int k = t; k < K; k += kThreads) {
      otok[k] = -1;
      onode[k] = -1;
    }
    if (t == 0) *alen = -1;
    return;
  }
  // A node's first child is tested against the target distribution itself
  // (nothing rejected yet), so that test too depends on the tree alone:
  // thread u takes it for node u, with the arithmetic of the walk's own
  // test below, and the walk then follows passing first children with one
  // read per node.
  if (t < n) {
    const int i = t;
    int c = -1;
#pragma unroll
    for (int w = kMaxSampledNodes / 32 - 1; w >= 0; --w)
      if (sh.kids[i][w]) c = 32 * w + __builtin_ctz(sh.kids[i][w]);
    if (c >= 0) {
      const float4 st = sh.kid_st[i];
      const float ip = 1.f / st.y, iq = 1.f / st.w;
      const float pt = exp2f((sh.kid_p[c] - st.x) * kLog2e) * ip;
      const float qt = exp2f((sh.kid_q[c] - st.z) * kLog2e) * iq;
      if (!(sh.kid_u[c] * qt < pt)) c = -1;
    }
    sh.fwd[i] = c;
  }
  __syncthreads();

  int u = 0, len = 1;  // current node, path length
  if (t == 0) sh.path[0] = 0;
  while (true) {
    for (int v; (v = __builtin_amdgcn_readfirstlane(sh.fwd[u])) >= 0; u = v) {
      if (t == 0) {
        sh.out[len - 1] = sh.token[v];
        sh.path[len] = v;
      }
      ++len;
    }
    const char *prow = (const char *)a.target_logits + ((int64_t)(base + u) * a.row_stride) * ESZ;
    const char *qrow = (const char *)a.draft_logits + ((int64_t)(base + u) * a.row_stride) * ESZ;
    uint32_t kids[kMaxSampledNodes / 32];
#pragma unroll
    for (int w = 0; w < kMaxSampledNodes / 32; ++w) kids[w] = __builtin_amdgcn_readfirstlane(sh.kids[u][w]);
    // the lowest child above c (-1: none), the first child, the last child
    auto next_kid = [&](int c) {
#pragma unroll
      for (int w = 0; w < kMaxSampledNodes / 32; ++w) {
        const int lo = c + 1 - 32 * w;  // first eligible bit of word w
        const uint32_t m = lo <= 0 ? kids[w] : lo >= 32 ? 0u : kids[w] & ~((1u << lo) - 1u);
        if (m) return 32 * w + __builtin_ctz(m);
      }
      return -1;
    };
    const int first_child = next_kid(-1);
    int last_child = -1;
#pragma unroll
    for (int w = 0; w < kMaxSampledNodes / 32; ++w)
      if (kids[w]) last_child = 32 * w + 31 - __builtin_clz(kids[w]);
    const float4 st = sh.kid_st[u];
    Residual R;
    R.mp = st.x;
    R.ip = 1.f / st.y;
    R.has_q = first_child >= 0;
    R.mq = st.z;
    R.iq = 1.f / st.w;
    R.c = 0.f;
    float S = 1.f;  // mass of the current residual (exactly 1 for p itself)
    int next = -1;
    bool after_last = false;  // the last child was rejected: draw from its residual R2
    Residual R2 = R;
    for (int c = first_child; c >= 0; c = next_kid(c)) {
      const float pt = exp2f((sh.kid_p[c] - R.mp) * kLog2e) * R.ip;
      const float qt = exp2f((sh.kid_q[c] - R.mq) * kLog2e) * R.iq;
      const float rt = (R.c == 0.f ? pt : fmaxf(pt - R.c * qt, 0.f)) / S;
      if (sh.kid_u[c] * qt < rt) {
        next = c;
        break;
      }
      R2 = R;
      R2.c = R.c + S;
      // After the last child no acceptance test needs the new mass: the
      // draw's own pass sums the same residual (no separate pass here)
      if (c == last_child) {
        after_last = true;
        break;
      }
      const float S2 = residual_mass<BF16>(prow, qrow, a.vocab, R2, sh);
      if (!(S2 > 0.f)) break;  // no mass left (rounding): draw from the residual before it
      R = R2;
      S = S2;
    }
    if (next < 0) {
      // After the last child, draw from R2; -1 means that rejection left no
      // mass (a sum of non-negative terms is zero only when every term is),
      // and the draw is taken from the residual before it (one call site,
      // so the draw's code is not inlined twice)
      int v = -1;
      for (int attempt = after_last ? 0 : 1; attempt < 2 && v < 0; ++attempt)
        v = residual_draw<BF16>(prow, qrow, a.vocab, attempt == 0 ? R2 : R, a.u_bonus[base + u],
                                a.stats + (int64_t)(base + u) * a.stats_parts, a.stats_sub, sh);
      if (t == 0) sh.out[len - 1] = v;
      break;
    }
    if (t == 0) {
      sh.out[len - 1] = sh.token[next];
      sh.path[len] = next;
    }
    ++len;
    u = next;
  }
  __syncthreads();
  for (int k = t; k < K; k += kThreads) {
    otok[k] = k < len ? sh.out[k] : -1;
    onode[k] = k < len ? sh.path[k] : -1;
  }
  if (t == 0) *alen = len;
}

}  // namespace

hipError_t launch_sampled_accept(const SampledArgs &a, bool bf16, hipStream_t stream) {
  if (a.num_requests == 0) return hipSuccess;
  if (a.total_nodes > 0) {
    const dim3 grid((unsigned)(a.total_nodes * a.stats_parts)), block(kStatsThreads);
    if (bf16)
      hipLaunchKernelGGL(sampled_stats_kernel<true>, grid, block, 0, stream, a);
    else
      hipLaunchKernelGGL(sampled_stats_kernel<false>, grid, block, 0, stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (bf16)
    hipLaunchKernelGGL(sampled_accept_kernel<true>, dim3((unsigned)a.num_requests), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(sampled_accept_kernel<false>, dim3((unsigned)a.num_requests), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace adaserve
