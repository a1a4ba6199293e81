// Per-node vocabulary argmax of the verification logits on gfx950.
//
// After verification the logits of every tree node give the target model's
// choice at that node (section 5.1); under greedy verification that choice
// is the row's highest-scoring token.  The scan is a pure HBM stream: one
// workgroup per row, every lane issuing 16-byte loads, several in flight,
// then a wave/workgroup reduction of (value, index) pairs in which the
// larger value wins and equal values keep the lower index.  Batches with at
// most one row per CU get 16-wave workgroups, so that more loads are in
// flight.
#include <limits.h>

#include "device_common.h"
#include "kernels.h"

namespace adaserve {

namespace {

constexpr int kUnroll = 8;
constexpr int kRowsForWide = 256;  // one row per CU

__device__ __forceinline__ void take_if_better(float v, int i, float &best, int &bi) {
  if (v > best || (v == best && i < bi)) {
    best = v;
    bi = i;
  }
}

// Strict greater-than update: used where indices visited by one lane only
// increase, so the first occurrence of the lane's maximum is kept.
__device__ __forceinline__ void take_if_greater(float v, int i, float &best, int &bi) {
  const bool gt = v > best;
  best = gt ? v : best;
  bi = gt ? i : bi;
}

template <bool BF16>
__device__ __forceinline__ float load_scalar(const void *p, int64_t i) {
  if (BF16) return bf16_bits_to_float(((const uint16_t *)p)[i]);
  return ((const float *)p)[i];
}

template <bool BF16>
__device__ __forceinline__ void scan_vector(const u32x4 &w, int idx0, float &best, int &bi) {
  if (BF16) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      take_if_greater(__uint_as_float(w[k] << 16), idx0 + 2 * k, best, bi);
      take_if_greater(__uint_as_float(w[k] & 0xffff0000u), idx0 + 2 * k + 1, best, bi);
    }
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) take_if_greater(__uint_as_float(w[k]), idx0 + k, best, bi);
  }
}

template <bool BF16, int kThreads>
__global__ __launch_bounds__(kThreads) void node_argmax_kernel(const void *logits, int64_t row_stride,
                                                              int32_t rows, int32_t vocab,
                                                              int32_t *out) {
  constexpr int ESZ = BF16 ? 2 : 4;
  constexpr int EPV = 16 / ESZ;  // elements per 16-byte vector
  const int row = blockIdx.x;
  if (row >= rows) return;
  const int tid = threadIdx.x;
  const char *p = (const char *)logits + (int64_t)row * row_stride * ESZ;
  float best = -INFINITY;
  int bi = INT_MAX;

  // Unaligned head (scalar), then 16-byte vectors, then the scalar tail.
  const uintptr_t addr = (uintptr_t)p;
  const int head = min((int)(((16 - (addr & 15)) & 15) / ESZ), vocab);
  if (tid < head) take_if_greater(load_scalar<BF16>(p, tid), tid, best, bi);
  const int nvec = (vocab - head) / EPV;
  const u32x4 *vp = (const u32x4 *)(p + (int64_t)head * ESZ);
  int i = tid;
  for (; i + (kUnroll - 1) * kThreads < nvec; i += kUnroll * kThreads) {
    u32x4 w[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) w[u] = __builtin_nontemporal_load(vp + i + u * kThreads);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) scan_vector<BF16>(w[u], head + (i + u * kThreads) * EPV, best, bi);
  }
  for (; i < nvec; i += kThreads) scan_vector<BF16>(vp[i], head + i * EPV, best, bi);
  for (int j = head + nvec * EPV + tid; j < vocab; j += kThreads)
    take_if_greater(load_scalar<BF16>(p, j), j, best, bi);

  // Reduce (value, index) over the wave, then over the workgroup.
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(best, off, 64);
    const int oi = __shfl_xor(bi, off, 64);
    take_if_better(ov, oi, best, bi);
  }
  __shared__ float sv[kThreads / 64];
  __shared__ int si[kThreads / 64];
  if ((tid & 63) == 0) {
    sv[tid >> 6] = best;
    si[tid >> 6] = bi;
  }
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < kThreads / 64; ++w) take_if_better(sv[w], si[w], best, bi);
    out[row] = (bi >= 0 && bi < vocab) ? bi : 0;  // all-NaN row: index 0
  }
}

template <bool BF16, int kThreads>
hipError_t launch_width(const void *logits, int64_t row_stride, int32_t rows, int32_t vocab, int32_t *out,
                        hipStream_t stream) {
  hipLaunchKernelGGL((node_argmax_kernel<BF16, kThreads>), dim3((unsigned)rows), dim3(kThreads), 0, stream,
                     logits, row_stride, rows, vocab, out);
  return hipGetLastError();
}

// 16 waves per row when the batch has at most one row per CU (measured on
// the 256-row long-context batch: 21 us instead of 24 us), else 4 waves
// (wider workgroups measured slower on 576 rows and more).
template <bool BF16>
hipError_t launch_rows(const void *logits, int64_t row_stride, int32_t rows, int32_t vocab, int32_t *out,
                       hipStream_t stream) {
  if (rows <= kRowsForWide) return launch_width<BF16, 1024>(logits, row_stride, rows, vocab, out, stream);
  return launch_width<BF16, 256>(logits, row_stride, rows, vocab, out, stream);
}

}  // namespace

hipError_t launch_node_argmax(const void *logits, int64_t row_stride, int32_t rows, int32_t vocab,
                              bool bf16, int32_t *out, hipStream_t stream) {
  if (rows == 0) return hipSuccess;
  return bf16 ? launch_rows<true>(logits, row_stride, rows, vocab, out, stream)
              : launch_rows<false>(logits, row_stride, rows, vocab, out, stream);
}

}  // namespace adaserve
