// Accepted-path KV commit on gfx950: after acceptance, the keys and values of
// the accepted root..i* path move from the tree rows into the request's
// paged cache at positions L_r .. L_r + d*, so that the next iteration sees
// them as prefix (section 5.1: verified tokens are stored back into the
// request pool for the next iteration).
//
// One workgroup per request.  The rows to commit are known after one pass
// over them (the first row whose node, position or page is invalid ends the
// commit); then every thread copies 16-byte pieces of (row, kv-head) K and V
// with plain vector loads and stores.  The copy is HBM/latency bound and
// tiny next to attention: (d*+1) x Hkv x D x 2 tensors per request.
#include "device_common.h"
#include "kernels.h"

namespace adaserve {

namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void commit_kv_kernel(CommitArgs a) {
  __shared__ int32_t first_bad;
  const int r = blockIdx.x;
  if (r >= a.num_requests) return;
  const int tid = threadIdx.x;
  const int32_t len = a.accept_len[r];
  const int32_t L = a.prefix_len[r];
  const int32_t node_base = a.node_indptr[r];
  const int32_t n = a.node_indptr[r + 1] - node_base;
  const bool any = len >= 1 && len <= a.max_accept && L >= 0 && n >= 1;
  if (tid == 0) first_bad = any ? len : 0;
  __syncthreads();
  // Rows that cannot be committed: the first one ends the commit.
  if (any) {
    for (int k = tid; k < len; k += kThreads) {
      const int32_t node = a.accept_nodes[(int64_t)r * a.max_accept + k];
      const int64_t t = (int64_t)L + k;
      const int64_t e = t / a.page_size;
      bool ok = node >= 0 && node < n && e < a.bt_stride;
      if (ok) {
        const int32_t p = a.block_table[(int64_t)r * a.bt_stride + e];
        ok = p >= 0 && p < a.num_pages;
      }
      if (!ok) atomicMin(&first_bad, k);
    }
  }
  __syncthreads();
  const int32_t rows = first_bad;
  // Copy: work item = (row, kv-head, 16-byte piece), K then V.
  const int pieces = a.row_bytes / 16;  // per (row, kv-head)
  const int64_t per_row = (int64_t)a.num_kv_heads * pieces;
  const int64_t items = (int64_t)rows * per_row;
  for (int64_t w = tid; w < items; w += kThreads) {
    const int32_t k = (int32_t)(w / per_row);
    const int32_t rem = (int32_t)(w - (int64_t)k * per_row);
    const int32_t h = rem / pieces, piece = rem - h * pieces;
    const int32_t node = a.accept_nodes[(int64_t)r * a.max_accept + k];
    const int64_t t = (int64_t)L + k;
    const int32_t p = a.block_table[(int64_t)r * a.bt_stride + t / a.page_size];
    const int64_t src = (((int64_t)(node_base + node) * a.num_kv_heads + h) * a.row_bytes) + piece * 16;
    const int64_t dst = ((((int64_t)p * a.num_kv_heads + h) * a.page_size + t % a.page_size) * a.row_bytes) +
                        piece * 16;
    *(u32x4 *)((char *)a.k_pages + dst) = *(const u32x4 *)((const char *)a.k_tree + src);
    *(u32x4 *)((char *)a.v_pages + dst) = *(const u32x4 *)((const char *)a.v_tree + src);
  }
  // every thread has read prefix_len[r] before this write (the barrier above)
  if (tid == 0) a.new_prefix_len[r] = any ? L + rows : L;
}

}  // namespace

hipError_t launch_commit_kv(const CommitArgs &a, hipStream_t stream) {
  if (a.num_requests == 0) return hipSuccess;
  hipLaunchKernelGGL(commit_kv_kernel, dim3((unsigned)a.num_requests), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace adaserve
