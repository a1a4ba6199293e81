// Per-row vocabulary argmax (device code shared by the standalone argmax
// kernel and the fused verification step): the scan is a pure HBM stream,
// every lane issuing 16-byte loads with several in flight, then a
// wave/workgroup reduction of (value, index) pairs in which the larger value
// wins and equal values keep the lower index.
#pragma once
#include <limits.h>

#include "device_common.h"

namespace adaserve {

constexpr int kArgmaxUnroll = 8;

__device__ __forceinline__ void argmax_take_if_better(float v, int i, float &best, int &bi) {
  if (v > best || (v == best && i < bi)) {
    best = v;
    bi = i;
  }
}

// Strict greater-than update: used where indices visited by one lane only
// increase, so the first occurrence of the lane's maximum is kept.
__device__ __forceinline__ void argmax_take_if_greater(float v, int i, float &best, int &bi) {
  const bool gt = v > best;
  best = gt ? v : best;
  bi = gt ? i : bi;
}

template <bool BF16>
__device__ __forceinline__ float argmax_load_scalar(const void *p, int64_t i) {
  if (BF16) return bf16_bits_to_float(((const uint16_t *)p)[i]);
  return ((const float *)p)[i];
}

template <bool BF16>
__device__ __forceinline__ void argmax_scan_vector(const u32x4 &w, int idx0, float &best, int &bi) {
  if (BF16) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      argmax_take_if_greater(__uint_as_float(w[k] << 16), idx0 + 2 * k, best, bi);
      argmax_take_if_greater(__uint_as_float(w[k] & 0xffff0000u), idx0 + 2 * k + 1, best, bi);
    }
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) argmax_take_if_greater(__uint_as_float(w[k]), idx0 + k, best, bi);
  }
}

// out[row] = the lowest index of row `row`'s maximum over columns
// 0 .. vocab - 1, computed by the kThreads threads of the calling workgroup
// (all of them must call it).  sv / si: kThreads / 64 entries of LDS.
template <bool BF16, int kThreads>
__device__ __forceinline__ void argmax_row(const void *logits, int64_t row_stride, int32_t vocab, int32_t row,
                                           int32_t *out, float *sv, int *si) {
  constexpr int ESZ = BF16 ? 2 : 4;
  constexpr int EPV = 16 / ESZ;  // elements per 16-byte vector
  const int tid = threadIdx.x;
  const char *p = (const char *)logits + (int64_t)row * row_stride * ESZ;
  float best = -INFINITY;
  int bi = INT_MAX;

  // Unaligned head (scalar), then 16-byte vectors, then the scalar tail.
  const uintptr_t addr = (uintptr_t)p;
  const int head = min((int)(((16 - (addr & 15)) & 15) / ESZ), vocab);
  if (tid < head) argmax_take_if_greater(argmax_load_scalar<BF16>(p, tid), tid, best, bi);
  const int nvec = (vocab - head) / EPV;
  const u32x4 *vp = (const u32x4 *)(p + (int64_t)head * ESZ);
  int i = tid;
  for (; i + (kArgmaxUnroll - 1) * kThreads < nvec; i += kArgmaxUnroll * kThreads) {
    u32x4 w[kArgmaxUnroll];
#pragma unroll
    for (int u = 0; u < kArgmaxUnroll; ++u) w[u] = __builtin_nontemporal_load(vp + i + u * kThreads);
#pragma unroll
    for (int u = 0; u < kArgmaxUnroll; ++u)
      argmax_scan_vector<BF16>(w[u], head + (i + u * kThreads) * EPV, best, bi);
  }
  if (i < nvec) {
    // The last, partial batch: its loads still all go out together (one by
    // one they were waited for in turn); slots past the end reload the last
    // vector and are taken as -inf, which never replaces a lane's best.
    constexpr uint32_t kNegInf = BF16 ? 0xff80ff80u : 0xff800000u;
    u32x4 w[kArgmaxUnroll];
#pragma unroll
    for (int u = 0; u < kArgmaxUnroll; ++u) w[u] = __builtin_nontemporal_load(vp + min(i + u * kThreads, nvec - 1));
#pragma unroll
    for (int u = 0; u < kArgmaxUnroll; ++u) {
      const bool in = i + u * kThreads < nvec;
      argmax_scan_vector<BF16>(in ? w[u] : u32x4{kNegInf, kNegInf, kNegInf, kNegInf},
                               head + (in ? i + u * kThreads : 0) * EPV, best, bi);
    }
  }
  for (int j = head + nvec * EPV + tid; j < vocab; j += kThreads)
    argmax_take_if_greater(argmax_load_scalar<BF16>(p, j), j, best, bi);

  // Reduce (value, index) over the wave, then over the workgroup.
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(best, off, 64);
    const int oi = __shfl_xor(bi, off, 64);
    argmax_take_if_better(ov, oi, best, bi);
  }
  if ((tid & 63) == 0) {
    sv[tid >> 6] = best;
    si[tid >> 6] = bi;
  }
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < kThreads / 64; ++w) argmax_take_if_better(sv[w], si[w], best, bi);
    out[row] = (bi >= 0 && bi < vocab) ? bi : 0;  // all-NaN row: index 0
  }
}

}  // namespace adaserve
