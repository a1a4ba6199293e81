// Longest-accepted-path acceptance on gfx950: one wavefront per request
// (accept_wave.h).
#include "accept_wave.h"
#include "kernels.h"

namespace adaserve {

namespace {

__global__ __launch_bounds__(64) void tree_accept_kernel(int32_t num_requests, int32_t total_nodes,
                                                         const int32_t *indptr, const int32_t *parent,
                                                         const int32_t *draft, const int32_t *amax,
                                                         int32_t max_accept, int32_t *accept_len,
                                                         int32_t *accept_tokens, int32_t *accept_nodes) {
  __shared__ int32_t par[kMaxTreeNodes], dr[kMaxTreeNodes], am[kMaxTreeNodes];
  const int r = blockIdx.x;
  if (r >= num_requests) return;
  accept_request(r, total_nodes, indptr, parent, draft, amax, max_accept, accept_len, accept_tokens,
                 accept_nodes, par, dr, am);
}

}  // namespace

hipError_t launch_tree_accept(int32_t num_requests, int32_t total_nodes, const int32_t *indptr,
                              const int32_t *parent, const int32_t *draft, const int32_t *amax,
                              int32_t max_accept, int32_t *accept_len, int32_t *accept_tokens,
                              int32_t *accept_nodes, hipStream_t stream) {
  if (num_requests == 0) return hipSuccess;
  hipLaunchKernelGGL(tree_accept_kernel, dim3((unsigned)num_requests), dim3(64), 0, stream,
                     num_requests, total_nodes, indptr, parent, draft, amax, max_accept,
                     accept_len, accept_tokens, accept_nodes);
  return hipGetLastError();
}

}  // namespace adaserve
