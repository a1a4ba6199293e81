// Tree selection on gfx950: the SLO-customised and throughput-optimised
// selection phases of Algorithm 2 (section 4.3 steps 2 and 3), which turn
// every request's candidate token tree into the draft token tree that
// verification scores.
//
// The whole batch is one workgroup of 1024 threads with everything in LDS
// (at most 8192 candidates): each request's candidates (at most 127) are
// ranked by one wave with a bitonic network in registers on a 64-bit key
// (path probability descending, depth, index) and written to the request's
// contiguous best-first segment; one thread per request walks its segment
// adding path probabilities in float32 to find how many picks reach its
// need; one thread deals the budget to the
// requests in descending order of need; a second bitonic sort ranks the
// remaining candidates of the whole batch (probability descending, depth,
// request, index) and the first `remaining budget` of them are added.
// Ties go to the smaller depth, so a node is never picked before its parent
// and every tree stays connected (appendix: greedy selection is connected).
#include "device_common.h"
#include "kernels.h"

namespace adaserve {

namespace {

constexpr int kThreads = 1024;
constexpr uint64_t kNone = ~0ull;

// A NaN need asks for nothing and ranks last.
__device__ __forceinline__ float sane_need(float x) { return x != x ? -INFINITY : x; }

__device__ __forceinline__ void bitonic_sort(uint64_t *key, int n) {
  for (int k = 2; k <= n; k <<= 1)
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = threadIdx.x; i < n; i += kThreads) {
        const int ixj = i ^ j;
        if (ixj > i) {
          const uint64_t a = key[i], b = key[ixj];
          const bool up = (i & k) == 0;
          if ((a > b) == up) {
            key[i] = b;
            key[ixj] = a;
          }
        }
      }
      __syncthreads();
    }
}

__global__ __launch_bounds__(kThreads) void select_trees_kernel(SelectArgs a) {
  __shared__ uint64_t key[kSelectMaxCandidates];
  __shared__ float prob[kSelectMaxCandidates];
  __shared__ int16_t par[kSelectMaxCandidates];
  __shared__ uint8_t depth[kSelectMaxCandidates];
  __shared__ uint8_t picked[kSelectMaxCandidates];
  __shared__ int32_t lo[kSelectMaxRequests + 1];
  __shared__ int32_t ok[kSelectMaxRequests];
  __shared__ int32_t seg[kSelectMaxRequests];     // start of the request's sorted segment
  __shared__ int32_t want[kSelectMaxRequests];    // SLO picks before the budget
  __shared__ int32_t take[kSelectMaxRequests];    // SLO picks granted
  __shared__ int32_t order[kSelectMaxRequests];   // requests by descending need
  __shared__ int32_t batch_ok, remaining;

  const int tid = threadIdx.x;
  const int B = a.num_requests, C = a.num_candidates;
  if (tid == 0) batch_ok = 1;
  for (int r = tid; r <= B; r += kThreads) lo[r] = a.cand_indptr[r];
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
  __syncthreads();
  auto request_of = [&](int i) {   // the r with lo[r] <= i < lo[r + 1] (lo is sorted here)
    int l = 0, h = B - 1;
    while (l < h) {
      const int m = (l + h + 1) >> 1;
      if (lo[m] <= i) l = m; else h = m - 1;
    }
    return l;
  };
  if (good)
    for (int i = tid; i < C; i += kThreads) {
      const int r = request_of(i);
      const int local = i - lo[r];
      const int p = par[i];
      const float f = prob[i];
      bool valid = p == -1 || (p >= 0 && p < local);
      if (valid) {
        const float fp = p == -1 ? 1.f : prob[lo[r] + p];
        valid = f > 0.f && f <= fp;   // NaN fails
      }
      if (!valid) ok[r] = 0;
    }
  __syncthreads();
  // depths (a walk up the parents; well-formed requests only)
  if (good)
    for (int i = tid; i < C; i += kThreads) {
      const int r = request_of(i);
      int d = 0;
      if (ok[r]) {
        int v = i - lo[r];
        while (v >= 0) {
          ++d;
          v = par[lo[r] + v];
        }
      }
      depth[i] = (uint8_t)d;
    }
  // segment starts: well-formed requests in index order
  if (tid == 0) {
    int s = 0;
    for (int r = 0; r < B; ++r) {
      seg[r] = s;
      if (ok[r]) s += lo[r + 1] - lo[r];
    }
  }
  __syncthreads();
  // sort 1, per request: (probability descending, depth, index); one wave
  // sorts a request's (at most 127) keys in registers, two per lane, with a
  // bitonic network, and writes them to the request's segment
  {
    const int lane = tid & 63, wave = tid >> 6;
    for (int r = wave; r < B; r += kThreads / 64) {
      if (!ok[r]) continue;
      const int nr = lo[r + 1] - lo[r];
      uint64_t k2[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int j = lane + 64 * h;
        const int i = lo[r] + j;
        k2[h] = j < nr ? ((uint64_t)(~__float_as_uint(prob[i])) << 23) | ((uint64_t)depth[i] << 16) |
                             ((uint64_t)j << 9)
                       : kNone;
      }
      for (int k = 2; k <= 128; k <<= 1)
        for (int j = k >> 1; j > 0; j >>= 1) {
          uint64_t nk[2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int e = lane + 64 * h;   // element index; its partner is e ^ j
            const uint64_t other = j == 64 ? k2[h ^ 1] : (uint64_t)__shfl_xor((unsigned long long)k2[h], j, 64);
            const bool lower = (e & j) == 0;
            const bool up = (e & k) == 0;   // ascending block
            const uint64_t mn = other < k2[h] ? other : k2[h], mx = other < k2[h] ? k2[h] : other;
            nk[h] = (lower == up) ? mn : mx;
          }
          k2[0] = nk[0];
          k2[1] = nk[1];
        }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int j = lane + 64 * h;
        if (j < nr) key[seg[r] + j] = k2[h];
      }
    }
  }
  __syncthreads();

  // each request's SLO picks: add the best remaining candidate while the
  // float32 sum of the added probabilities is below its need and the tree is
  // under n_max nodes
  for (int r = tid; r < B; r += kThreads) {
    int k = 0;
    if (ok[r]) {
      const int nr = lo[r + 1] - lo[r];
      const float need = sane_need(a.need[r]);
      float acc = 0.f;
      while (k < nr && acc < need && 1 + k < a.n_max) {
        acc += __uint_as_float(~(uint32_t)(key[seg[r] + k] >> 23));
        ++k;
      }
    }
    want[r] = k;
  }
  // requests by descending need, ties by index
  for (int r = tid; r < B; r += kThreads) {
    if (!ok[r]) continue;
    const float nr = sane_need(a.need[r]);
    int rank = 0;
    for (int q = 0; q < B; ++q) {
      if (!ok[q]) continue;
      const float nq = sane_need(a.need[q]);
      rank += (nq > nr || (nq == nr && q < r)) ? 1 : 0;
    }
    order[rank] = r;
  }
  __syncthreads();
  if (tid == 0) {
    int valid = 0;
    for (int r = 0; r < B; ++r) {
      valid += ok[r] ? 1 : 0;
      take[r] = 0;
    }
    int left = a.budget - valid;
    for (int k = 0; k < valid; ++k) {
      const int r = order[k];
      const int t = min(want[r], max(left, 0));
      take[r] = t;
      left -= t;
    }
    remaining = max(left, 0);
  }
  __syncthreads();
  for (int r = tid; r < B; r += kThreads)
    for (int k = 0; k < take[r]; ++k) {
      const int local = (int)((key[seg[r] + k] >> 9) & 0x7f);
      picked[lo[r] + local] = 1;
    }
  __syncthreads();

  // sort 2: the remaining candidates of the batch, best first
  int n = 2;
  while (n < C) n <<= 1;
  for (int i = tid; i < n; i += kThreads) {
    uint64_t k = kNone;
    if (good && i < C && !picked[i]) {
      const int r = request_of(i);
      if (ok[r])
        k = ((uint64_t)(~__float_as_uint(prob[i])) << 32) | ((uint64_t)depth[i] << 25) |
            ((uint64_t)r << 16) | (uint64_t)(i - lo[r]);
    }
    key[i] = k;
  }
  __syncthreads();
  bitonic_sort(key, n);
  for (int k = tid; k < remaining && k < n; k += kThreads) {
    const uint64_t kk = key[k];
    if (kk == kNone) continue;
    const int r = (int)((kk >> 16) & 0x1ff), local = (int)(kk & 0x7f);
    picked[lo[r] + local] = 1;
  }
  __syncthreads();

  // output: root first, then the picked candidates by (depth, index)
  int16_t *tree_id = (int16_t *)key;   // key[] is free now
  if (good)
    for (int i = tid; i < C; i += kThreads) {
      const int r = request_of(i);
      int16_t t = -1;
      if (ok[r] && picked[i]) {
        int before = 0;
        for (int j = lo[r]; j < lo[r + 1]; ++j)
          before += (picked[j] && (depth[j] < depth[i] || (depth[j] == depth[i] && j < i))) ? 1 : 0;
        t = (int16_t)(1 + before);
      }
      tree_id[i] = t;
    }
  __syncthreads();
  for (int w = tid; w < B * a.max_nodes; w += kThreads) {
    a.tree_parent[w] = -1;
    a.tree_cand[w] = -1;
  }
  __syncthreads();   // the row fills above happen before the entries below
  if (good)
    for (int i = tid; i < C; i += kThreads) {
      const int t = tree_id[i];
      if (t < 0) continue;
      const int r = request_of(i);
      const int p = par[i];
      a.tree_cand[(int64_t)r * a.max_nodes + t] = i - lo[r];
      a.tree_parent[(int64_t)r * a.max_nodes + t] = p == -1 ? 0 : tree_id[lo[r] + p];
    }
  for (int r = tid; r < B; r += kThreads) {
    int cnt = 0;
    if (ok[r])
      for (int j = lo[r]; j < lo[r + 1]; ++j) cnt += picked[j];
    a.tree_size[r] = ok[r] ? 1 + cnt : -1;
  }
}

}  // namespace

hipError_t launch_select_trees(const SelectArgs &a, hipStream_t stream) {
  if (a.num_requests == 0) return hipSuccess;
  hipLaunchKernelGGL(select_trees_kernel, dim3(1), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace adaserve
