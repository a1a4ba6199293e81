// Accepted-path KV commit on gfx950: after acceptance, the keys and values of
// the accepted root..i* path move from the tree rows into the request's
// paged cache at positions L_r .. L_r + d*, so that the next iteration sees
// them as prefix (section 5.1: once verified, a request's tokens return with
// it to the pool of requests that the next iteration draws from).
//
// One workgroup per request, three rounds of dependent loads: the request's
// scalars; every path row's node and page at once (kept in LDS; the first
// row whose node, position or page is invalid ends the commit); then every
// thread copies 16-byte pieces of (row, kv-head) K and V.  The copy is
// latency bound and tiny next to attention: (d*+1) x Hkv x D x 2 per request.
#include "device_common.h"
#include "kernels.h"
#include "plan.h"

namespace adaserve {

namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void commit_kv_kernel(CommitArgs a) {
  __shared__ int32_t first_bad;
  __shared__ int64_t src_row[kMaxTreeNodes];   // global tree row of path row k
  __shared__ int64_t dst_cell[kMaxTreeNodes];  // page * page_size + slot of cache position L + k
  const int r = blockIdx.x;
  if (r >= a.num_requests) return;
  const int tid = threadIdx.x;
  // one round of loads for the request's scalars
  const int32_t len = a.accept_len[r];
  const int32_t L = a.prefix_len[r];
  const int32_t node_base = a.node_indptr[r];
  const int32_t n = a.node_indptr[r + 1] - node_base;
  const bool any = len >= 1 && len <= a.max_accept && len <= kMaxTreeNodes && L >= 0 && n >= 1;
  if (tid == 0) first_bad = any ? len : 0;
  __syncthreads();
  // one round for the path rows and their pages; the first row that cannot
  // be committed ends the commit
  if (any && tid < len) {
    const int k = tid;
    const int32_t node = a.accept_nodes[(int64_t)r * a.max_accept + k];
    const int64_t t = (int64_t)L + k;
    const int64_t e = t / a.page_size;
    const int32_t p = e < a.bt_stride ? a.block_table[(int64_t)r * a.bt_stride + e] : -1;
    const bool ok = node >= 0 && node < n && p >= 0 && p < a.num_pages;
    src_row[k] = (int64_t)node_base + node;
    dst_cell[k] = (int64_t)p * a.page_size + t % a.page_size;
    if (!ok) atomicMin(&first_bad, k);
  }
  __syncthreads();
  const int32_t rows = first_bad;
  // the copy: work item = (row, kv-head, 16-byte piece), K and V
  const int pieces = a.row_bytes / 16;  // per (row, kv-head)
  const int64_t per_row = (int64_t)a.num_kv_heads * pieces;
  const int64_t items = (int64_t)rows * per_row;
  for (int64_t w = tid; w < items; w += kThreads) {
    const int32_t k = (int32_t)(w / per_row);
    const int32_t rem = (int32_t)(w - (int64_t)k * per_row);
    const int32_t h = rem / pieces, piece = rem - h * pieces;
    const int64_t cell = dst_cell[k];
    const int64_t page = cell / a.page_size, slot = cell - page * a.page_size;
    const int64_t src = (src_row[k] * a.num_kv_heads + h) * a.row_bytes + piece * 16;
    const int64_t dst = ((page * a.num_kv_heads + h) * a.page_size + slot) * a.row_bytes + piece * 16;
    *(u32x4 *)((char *)a.k_pages + dst) = *(const u32x4 *)((const char *)a.k_tree + src);
    *(u32x4 *)((char *)a.v_pages + dst) = *(const u32x4 *)((const char *)a.v_tree + src);
  }
  // every thread read prefix_len[r] before the first barrier
  if (tid == 0) a.new_prefix_len[r] = any ? L + rows : L;
}

}  // namespace

hipError_t launch_commit_kv(const CommitArgs &a, hipStream_t stream) {
  if (a.num_requests == 0) return hipSuccess;
  hipLaunchKernelGGL(commit_kv_kernel, dim3((unsigned)a.num_requests), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace adaserve
