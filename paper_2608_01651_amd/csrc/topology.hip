// Tree topology export: the M+ rows (inclusive ancestor masks) and depths that
// the verify kernel builds on chip (§4.1 notation table; built once per
// request per round and reusable across layers and heads, §4.3).  One
// workgroup per request, one thread per node, pointer jumping as in verify.
#include <hip/hip_runtime.h>

#include "tl_device.h"
#include "tl_kernels.h"

namespace tl {

__global__ __launch_bounds__(kThreads) void topology_kernel(TopoArgs a) {
  __shared__ int s_jmp[kThreads];
  __shared__ float s_acc[kThreads];
  __shared__ int s_cnt[kThreads];
  __shared__ uint64_t s_msk[4 * kThreads];
  const int tid = threadIdx.x;
  Request rq;
  if (!load_request(a.node_offsets, blockIdx.x, a.max_nodes, a.dev_err, rq)) return;
  if (rq.T == 0) return;
  int dep;
  float cl;
  uint64_t msk[4];
  const int par = (tid < rq.T) ? a.parent[rq.off + tid] : -1;
  if (!build_topology<4, true>(par, rq.T, 0.f, s_jmp, s_acc, s_cnt, s_msk, dep, cl, msk)) {
    if (tid == 0) report(a.dev_err, TL_EBADTREE);
    return;
  }
  if (tid < rq.T) {
    const size_t r = (size_t)(rq.off + tid);
    a.depth[r] = dep;
#pragma unroll
    for (int w = 0; w < 4; ++w)
      if (w < a.words) a.anc_mask[r * a.words + w] = msk[w];
  }
}

tl_status launch_topology(const TopoArgs& a, hipStream_t stream) {
  if (a.batch == 0) return TL_OK;
  hipLaunchKernelGGL(topology_kernel, dim3((unsigned)a.batch), dim3(kThreads), 0, stream, a);
  return hipGetLastError() == hipSuccess ? TL_OK : TL_EHIP;
}

}  // namespace tl
