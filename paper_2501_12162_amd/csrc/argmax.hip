// Per-node vocabulary argmax of the verification logits on gfx950.
//
// After verification the logits of every tree node give the target model's
// choice at that node (section 5.1); under greedy verification that choice
// is the row's highest-scoring token.  One workgroup per row (argmax_row.h);
// batches with at most one row per CU get 16-wave workgroups, so that more
// loads are in flight.
#include "argmax_row.h"
#include "kernels.h"

namespace adaserve {

namespace {

constexpr int kRowsForWide = 256;  // one row per CU

template <bool BF16, int kThreads>
__global__ __launch_bounds__(kThreads) void node_argmax_kernel(const void *logits, int64_t row_stride,
                                                              int32_t rows, int32_t vocab,
                                                              int32_t *out) {
  __shared__ float sv[kThreads / 64];
  __shared__ int si[kThreads / 64];
  const int row = blockIdx.x;
  if (row >= rows) return;
  argmax_row<BF16, kThreads>(logits, row_stride, vocab, row, out, sv, si);
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
