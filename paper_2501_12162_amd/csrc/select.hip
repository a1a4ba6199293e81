// Tree selection on gfx950: the SLO-customised and throughput-optimised
// selection phases of Algorithm 2 (section 4.3 steps 2 and 3), which turn
// every request's candidate token tree into the draft token tree that
// verification scores.
//
// The whole batch is one workgroup of 1024 threads with everything in LDS
// (at most 8192 candidates):
// * each candidate gets a 55-bit key (path probability descending, depth,
//   index) and finds its place in its request's best-first order by counting
//   the request's keys below it (at most 127 broadcast LDS reads);
// * one thread per request walks its ordered segment adding path
//   probabilities in float32 to find how many picks reach its need;
// * the budget is dealt in descending order of need as a prefix sum: a
//   request is granted what is left after the wants of every request ranked
//   before it;
// * the throughput phase needs only the best `remaining budget` of the
//   candidates left over (probability descending, depth, request, index):
//   a radix select over 11-bit digits of the keys, held in registers, finds
//   the threshold key, stopping as soon as the digit bucket it lands in is
//   taken whole;
// * one wave per request numbers the picked candidates by (depth, index)
//   with ballots and writes the request's output rows.
// Ties go to the smaller depth, so a node is never picked before its parent
// and every tree stays connected (appendix: greedy selection is connected).
#include "device_common.h"
#include "kernels.h"

namespace adaserve {

namespace {

constexpr int kThreads = 1024;
constexpr int kPerThread = kSelectMaxCandidates / kThreads;
constexpr uint64_t kNone = ~0ull;
constexpr int kDigitBits = 11;
constexpr int kBins = 1 << kDigitBits;
constexpr int kTopShift = 44;   // keys are 55 bits: digits at 44, 33, 22, 11, 0

static_assert(kSelectMaxCandidates % kThreads == 0, "candidates per thread");
static_assert(kSelectMaxRequests <= 512 && kSelectMaxPerRequest <= 127, "key field widths");
static_assert(kBins * 4 <= kSelectMaxCandidates * 4, "the histogram lives in the probability array");

// A NaN need asks for nothing and ranks last.
__device__ __forceinline__ float sane_need(float x) { return x != x ? -INFINITY : x; }

// ~probability bits: a larger positive float gives a smaller value
__device__ __forceinline__ uint64_t prob_desc(float p) { return (uint64_t)(~__float_as_uint(p)); }

__global__ __launch_bounds__(kThreads) void select_trees_kernel(SelectArgs a) {
  __shared__ __align__(16) uint64_t key[kSelectMaxCandidates];   // request segments, best first
  __shared__ float prob[kSelectMaxCandidates];     // later the radix histogram
  __shared__ int16_t par[kSelectMaxCandidates];
  __shared__ uint16_t rq[kSelectMaxCandidates];    // request of each candidate
  __shared__ uint8_t depth[kSelectMaxCandidates];
  __shared__ uint8_t picked[kSelectMaxCandidates];
  __shared__ int32_t lo[kSelectMaxRequests + 1];
  __shared__ int32_t ok[kSelectMaxRequests];
  __shared__ int2 wn[kSelectMaxRequests];          // (SLO picks before the budget or -1, need bits)
  __shared__ int32_t take[kSelectMaxRequests];     // SLO picks granted
  __shared__ int32_t batch_ok, remaining;
  __shared__ int32_t sel_digit, sel_rank, sel_count, sel_all;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int B = a.num_requests, C = a.num_candidates;
  if (tid == 0) batch_ok = 1;
  for (int r = tid; r <= B; r += kThreads) lo[r] = a.cand_indptr[r];
  for (int r = tid; r < B; r += kThreads) wn[r] = make_int2(-1, __float_as_int(sane_need(a.need[r])));
  __syncthreads();
  // the index array must describe exactly the C candidates
  for (int r = tid; r < B; r += kThreads)
    if (lo[r] > lo[r + 1]) batch_ok = 0;
  if (tid == 0 && (lo[0] != 0 || lo[B] != C)) batch_ok = 0;
  __syncthreads();
  const bool good = batch_ok != 0;

  // candidates into LDS; a request is well formed when it has at most 127
  // candidates, parents are -1 or earlier candidates, and path
  // probabilities lie in (0, 1] and never exceed the parent's
  for (int r = tid; r < B; r += kThreads) ok[r] = good && (lo[r + 1] - lo[r] <= kSelectMaxPerRequest);
  for (int i = tid; i < C; i += kThreads) {
    prob[i] = good ? a.cand_prob[i] : 0.f;
    par[i] = good ? (int16_t)max(-2, min(a.cand_parent[i], 32767)) : (int16_t)-2;
    picked[i] = 0;
  }
  if (good)   // the segments of a well-formed index array tile [0, C)
    for (int r = wave; r < B; r += kThreads / 64)
      for (int i = lo[r] + lane; i < lo[r + 1]; i += 64) rq[i] = (uint16_t)r;
  __syncthreads();
  if (good)
    for (int i = tid; i < C; i += kThreads) {
      const int r = rq[i];
      const int p = par[i];
      const float f = prob[i];
      bool valid = p == -1 || (p >= 0 && p < i - lo[r]);
      if (valid) {
        const float fp = p == -1 ? 1.f : prob[lo[r] + p];
        valid = f > 0.f && f <= fp;   // NaN fails
      }
      if (!valid) ok[r] = 0;
    }
  __syncthreads();
  // depths (a walk up the parents) and the request-local keys
  if (good)
    for (int i = tid; i < C; i += kThreads) {
      const int r = rq[i];
      uint64_t k = kNone;
      if (ok[r]) {
        int d = 0;
        for (int v = i - lo[r]; v >= 0; v = par[lo[r] + v]) ++d;
        depth[i] = (uint8_t)d;
        k = (prob_desc(prob[i]) << 23) | ((uint64_t)d << 16) | ((uint64_t)(i - lo[r]) << 9);
      }
      key[i] = k;
    }
  __syncthreads();

  // best-first order inside each request, one wave per request: a key's
  // place is the number of the request's keys below it (keys are distinct:
  // the index is part of them); the wave reads the whole segment before it
  // writes it back in order
  for (int r = wave; r < B; r += kThreads / 64) {
    const int base = lo[r], nr = lo[r + 1] - base;
    if (!ok[r] || nr == 0) continue;
    const uint64_t m0 = lane < nr ? key[base + lane] : kNone;
    const uint64_t m1 = lane + 64 < nr ? key[base + lane + 64] : kNone;
    // keys two at a time from 16-byte-aligned pairs, two counters per key
    int b0 = 0, b1 = 0, c0 = 0, c1 = 0;
    const int head = base & 1, pairs = (nr - head) >> 1;
    const ulonglong2 *kp = (const ulonglong2 *)(key + base + head);
    if (head) {
      const uint64_t kq = key[base];
      b0 += kq < m0 ? 1 : 0;
      b1 += kq < m1 ? 1 : 0;
    }
    if ((nr - head) & 1) {
      const uint64_t kq = key[base + nr - 1];
      c0 += kq < m0 ? 1 : 0;
      c1 += kq < m1 ? 1 : 0;
    }
    if (nr <= 64) {
#pragma unroll 8
      for (int q = 0; q < pairs; ++q) {
        const ulonglong2 x = kp[q];
        b0 += x.x < m0 ? 1 : 0;
        c0 += x.y < m0 ? 1 : 0;
      }
    } else {
#pragma unroll 4
      for (int q = 0; q < pairs; ++q) {
        const ulonglong2 x = kp[q];
        b0 += x.x < m0 ? 1 : 0;
        c0 += x.y < m0 ? 1 : 0;
        b1 += x.x < m1 ? 1 : 0;
        c1 += x.y < m1 ? 1 : 0;
      }
    }
    b0 += c0;
    b1 += c1;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");   // every read above precedes the writes
    if (lane < nr) key[base + b0] = m0;
    if (lane + 64 < nr) key[base + b1] = m1;
  }
  __syncthreads();

  // each request's SLO picks: add the best remaining candidate while the
  // float32 sum of the added probabilities is below its need and the tree is
  // under n_max nodes (keys are read four ahead of the running sum)
  for (int r = tid; r < B; r += kThreads) {
    int k = 0;
    if (ok[r]) {
      const int lim = min(lo[r + 1] - lo[r], a.n_max - 1);
      const float nd = __int_as_float(wn[r].y);
      const uint64_t *seg = key + lo[r];
      float acc = 0.f;
      while (k < lim && acc < nd) {
        float f[4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
          f[u] = k + u < lim ? __uint_as_float(~(uint32_t)(seg[k + u] >> 23)) : 0.f;
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (k < lim && acc < nd) {
            acc += f[u];
            ++k;
          }
      }
    }
    if (ok[r]) wn[r].x = k;
  }
  __syncthreads();
  // the budget, dealt in descending order of need (ties by index): every
  // well-formed request keeps its root, then a request gets what is left
  // after the wants of the requests ranked before it; a group of G lanes
  // shares each request's pass over the batch
  {
    int G = 64;
    while (G > 1 && G * B > kThreads) G >>= 1;
    const int r = tid / G, j = tid % G;
    int valid = 0, ahead = 0, total = 0;
    int2 me = make_int2(-1, 0);
    if (r < B) {
      me = wn[r];
      const float nr = __int_as_float(me.y);
#pragma unroll 4
      for (int q = j; q < B; q += G) {
        const int2 x = wn[q];
        const float nq = __int_as_float(x.y);
        const int w = max(x.x, 0);
        valid += x.x >= 0 ? 1 : 0;
        total += w;
        ahead += (nq > nr || (nq == nr && q < r)) ? w : 0;
      }
    }
    for (int o = 1; o < G; o <<= 1) {   // groups are aligned inside a wave
      valid += __shfl_xor(valid, o, 64);
      total += __shfl_xor(total, o, 64);
      ahead += __shfl_xor(ahead, o, 64);
    }
    if (r < B && j == 0) {
      const int left = a.budget - valid;
      take[r] = me.x >= 0 ? min(me.x, max(left - ahead, 0)) : 0;
      if (r == 0) remaining = max(left - total, 0);
    }
  }
  __syncthreads();
  for (int i = tid; i < C; i += kThreads)
    if (good) {
      const int r = rq[i];
      if (ok[r] && i - lo[r] < take[r]) picked[lo[r] + (int)((key[i] >> 9) & 0x7f)] = 1;
    }
  __syncthreads();

  // throughput phase: the best `remaining` of the candidates left, keyed
  // (probability descending, depth, request, index), found by radix select
  uint64_t k2[kPerThread];
#pragma unroll
  for (int s = 0; s < kPerThread; ++s) {
    const int i = tid + s * kThreads;
    k2[s] = kNone;
    if (good && i < C && ok[rq[i]] && !picked[i]) {
      const int r = rq[i];
      k2[s] = (prob_desc(prob[i]) << 23) | ((uint64_t)depth[i] << 16) | ((uint64_t)r << 7) | (uint64_t)(i - lo[r]);
    }
  }
  __syncthreads();   // prob[] is the histogram from here on
  if (remaining > 0) {
    uint32_t *hist = (uint32_t *)prob;
    uint64_t prefix = 0;   // the digits chosen so far
    int want_rank = remaining, shift = kTopShift;
    for (;; shift -= kDigitBits) {
      for (int b = tid; b < kBins; b += kThreads) hist[b] = 0;
      __syncthreads();
#pragma unroll
      for (int s = 0; s < kPerThread; ++s)
        if (k2[s] != kNone && (k2[s] >> (shift + kDigitBits)) == (prefix >> (shift + kDigitBits)))
          atomicAdd(&hist[(k2[s] >> shift) & (kBins - 1)], 1u);
      __syncthreads();
      if (wave == 0) {
        // lane l holds bins [32 l, 32 l + 32); the bucket holding the
        // want_rank-th key is where the running count first reaches it
        uint32_t c[32];
        const uint4 *h4 = (const uint4 *)(hist + 32 * lane);
        uint32_t sum = 0;
#pragma unroll
        for (int v = 0; v < 8; ++v) {
          const uint4 x = h4[v];
          c[4 * v] = x.x;
          c[4 * v + 1] = x.y;
          c[4 * v + 2] = x.z;
          c[4 * v + 3] = x.w;
          sum += x.x + x.y + x.z + x.w;
        }
        uint32_t incl = sum;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const uint32_t y = __shfl_up(incl, o, 64);
          if (lane >= o) incl += y;
        }
        const uint32_t total = __shfl(incl, 63, 64);
        const uint32_t wr = (uint32_t)want_rank;
        if (wr > total) {
          if (lane == 0) sel_all = 1;
        } else {
          const unsigned long long hit = __ballot(incl >= wr);
          if (lane == __ffsll((long long)hit) - 1) {
            uint32_t cum = incl - sum;
            int digit = 0;
            uint32_t cnt = 0;
            bool found = false;
#pragma unroll
            for (int b = 0; b < 32; ++b)
              if (!found && cum + c[b] >= wr) {
                found = true;
                digit = 32 * lane + b;
                cnt = c[b];
              } else if (!found) {
                cum += c[b];
              }
            sel_all = 0;
            sel_digit = digit;
            sel_rank = (int)(wr - cum);
            sel_count = (int)cnt;
          }
        }
      }
      __syncthreads();
      if (sel_all) {
        prefix = kNone;   // fewer keys left than budget: take them all
        break;
      }
      prefix |= (uint64_t)sel_digit << shift;
      want_rank = sel_rank;
      // a bucket taken whole ends the search; the last digit is one key
      if (sel_count == want_rank || shift == 0) break;
    }
#pragma unroll
    for (int s = 0; s < kPerThread; ++s)
      if (k2[s] != kNone && (k2[s] >> shift) <= (prefix >> shift)) picked[tid + s * kThreads] = 1;
  }
  __syncthreads();

  // output, one wave per request: root first, then the picked candidates by
  // (depth, index), numbered level by level with ballots
  const unsigned long long below = (1ull << lane) - 1;
  for (int r = wave; r < B; r += kThreads / 64) {
    int32_t *tp = a.tree_parent + (int64_t)r * a.max_nodes;
    int32_t *tc = a.tree_cand + (int64_t)r * a.max_nodes;
    if (!ok[r]) {
      for (int t = lane; t < a.max_nodes; t += 64) {
        tp[t] = -1;
        tc[t] = -1;
      }
      if (lane == 0) a.tree_size[r] = -1;
      continue;
    }
    const int base = lo[r], nr = lo[r + 1] - base;
    bool pk[2];
    int dp[2], id[2] = {-1, -1};
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int e = lane + 64 * h;
      pk[h] = e < nr && picked[base + e];
      dp[h] = e < nr ? depth[base + e] : 0;
    }
    const int total = __popcll(__ballot(pk[0])) + __popcll(__ballot(pk[1]));
    int next = 1;
    for (int d = 1; next <= total && d <= kSelectMaxPerRequest; ++d) {
      const bool at0 = pk[0] && dp[0] == d, at1 = pk[1] && dp[1] == d;
      const unsigned long long m0 = __ballot(at0), m1 = __ballot(at1);
      if (at0) id[0] = next + __popcll(m0 & below);
      if (at1) id[1] = next + __popcll(m0) + __popcll(m1 & below);
      next += __popcll(m0) + __popcll(m1);
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int e = lane + 64 * h;
      const int pp = e < nr ? par[base + e] : -1;
      const int src = pp < 0 ? 0 : pp;
      const int x0 = __shfl(id[0], src & 63, 64), x1 = __shfl(id[1], src & 63, 64);
      if (pk[h] && id[h] > 0) {
        tc[id[h]] = e;
        tp[id[h]] = pp < 0 ? 0 : (src < 64 ? x0 : x1);
      }
    }
    for (int t = lane; t < a.max_nodes; t += 64)
      if (t == 0 || t > total) {
        tp[t] = -1;
        tc[t] = -1;
      }
    if (lane == 0) a.tree_size[r] = 1 + total;
  }
}

}  // namespace

hipError_t launch_select_trees(const SelectArgs &a, hipStream_t stream) {
  if (a.num_requests == 0) return hipSuccess;
  hipLaunchKernelGGL(select_trees_kernel, dim3(1), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace adaserve
