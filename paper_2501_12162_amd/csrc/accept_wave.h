// Longest-accepted-path acceptance of one request by one wavefront (device
// code shared by the standalone acceptance kernel and the fused verification
// step).
//
// The tree (<= 128 nodes) is copied to LDS; each lane walks the root paths
// of its two nodes to get their depth and whether every node on the path
// matches (draft token == target argmax at the parent); a wave-wide max over
// (depth, -id) of accepted nodes picks the deepest accepted node with the
// smallest id; lanes then write the path and its tokens.  Greedy tree
// verification per section 4.3 step 4, read with section 2 (root = last
// generated token) and Algorithm 2's count of the root as one accepted token.
#pragma once
#include "device_common.h"
#include "plan.h"

namespace adaserve {

__device__ __forceinline__ int wave_max_int(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = max(v, __shfl_xor(v, off, 64));
  return v;
}

// Orders this wave's LDS writes before its later LDS reads (a wave's LDS
// operations execute in order; this keeps the compiler from moving them).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Acceptance of request r by the calling wave (all 64 lanes); par, dr, am:
// kMaxTreeNodes entries of LDS each, owned by this wave.
__device__ __forceinline__ void accept_request(int r, int32_t total_nodes, const int32_t *indptr,
                                               const int32_t *parent, const int32_t *draft, const int32_t *amax,
                                               int32_t max_accept, int32_t *accept_len, int32_t *accept_tokens,
                                               int32_t *accept_nodes, int32_t *par, int32_t *dr, int32_t *am) {
  const int lane = threadIdx.x & 63;
  int32_t *tok_row = accept_tokens + (int64_t)r * max_accept;
  int32_t *node_row = accept_nodes + (int64_t)r * max_accept;

  const int32_t a0 = indptr[r], a1 = indptr[r + 1];
  const int32_t n = a1 - a0;
  bool ok = a0 >= 0 && a1 <= total_nodes && n >= 1 && n <= kMaxTreeNodes;
  if (ok) {
    for (int i = lane; i < n; i += 64) {
      par[i] = parent[a0 + i];
      dr[i] = draft[a0 + i];
      am[i] = amax[a0 + i];
    }
  }
  wave_lds_sync();
  int bad = 0;
  if (ok) {
    for (int i = lane; i < n; i += 64) {
      const int p = par[i];
      bad |= (i == 0) ? (p != -1) : (p < 0 || p >= i);
    }
  }
  ok = ok && wave_max_int(bad) == 0;

  // Depth and acceptance of every node; key = (depth << 8) | (255 - id).
  int deepest = 0, best = -1;
  if (ok) {
    for (int i = lane; i < n; i += 64) {
      int v = i, d = 0;
      bool acc = true;
      while (v != 0) {
        const int p = par[v];
        acc = acc && dr[v] == am[p];
        v = p;
        ++d;
      }
      deepest = max(deepest, d);
      if (acc) best = max(best, (d << 8) | (255 - i));
    }
  }
  deepest = wave_max_int(deepest);
  best = wave_max_int(best);
  ok = ok && deepest < max_accept;

  if (!ok) {
    for (int k = lane; k < max_accept; k += 64) {
      tok_row[k] = -1;
      node_row[k] = -1;
    }
    if (lane == 0) accept_len[r] = -1;
    return;
  }
  const int dstar = best >> 8;
  const int istar = 255 - (best & 255);
  for (int k = lane; k < max_accept; k += 64) {
    int node = -1, token = -1;
    if (k <= dstar) {
      int child = istar;  // path node at depth k+1 (or i* itself when k == d*)
      for (int s = 0; s < dstar - k - 1; ++s) child = par[child];
      node = (k == dstar) ? istar : par[child];
      token = (k == dstar) ? am[istar] : dr[child];
    }
    tok_row[k] = token;
    node_row[k] = node;
  }
  if (lane == 0) accept_len[r] = dstar + 1;
}

}  // namespace adaserve
