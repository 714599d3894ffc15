// Tree topology export: the M+ rows (inclusive ancestor masks) and depths of
// the notation table of §4.1, built once per request per round and reusable
// across layers and heads (§4.3).  One workgroup per request.
//
// Every verify kernel builds the topology on chip with one of four
// routines, and the export runs the routine that the verify kernel serving
// the same problem runs, so that the bits it returns are the bits that
// kernel masks its coefficients with:
//   kTopoWaveN  wave_topology_n, one wavefront, ballot + shuffle pointer
//               jumping: gated linear attention over node caps of <= 64
//               (bf16, d >= 32), the small-tree MFMA kernel;
//   kTopoLds    build_topology<W>, one thread per node: root-path walks
//               through the parents in LDS, finished by pointer jumping for
//               deep trees: the delta rule's tile walk (where its layout
//               fits LDS), and the vector path (fp32 inputs or d = 16), whose
//               own pass counts depths without masks;
//   kTopoGdn    the delta rule's kernel for node caps beyond the tile walk's
//               LDS (d = 128, caps of 176..256): wave_topology for trees of
//               <= 64 nodes, build_topology<4> above;
//   kTopoJump1  wave_topology_jump, one wavefront holding 64 W nodes
//               (pointer jumping in LDS, no workgroup barrier): the delta
//               rule's dense kernel (bf16, d = 128, node caps of up to 128)
//               and the large-tree kernel of gated linear attention (bf16,
//               d >= 32, caps of 65..256).
// The depth of a node is its number of strict ancestors; where the routine
// yields only the mask it is the mask's popcount minus one.
#include <hip/hip_runtime.h>

#include "tl_device.h"
#include "tl_kernels.h"
#include "verify_gla_small.h"

namespace tl {

enum TopoKind { kTopoWaveN = 0, kTopoLds = 1, kTopoGdn = 2, kTopoJump1 = 3 };

template <int W>
__device__ inline void store_topology(const TopoArgs& a, const Request& rq, int node, int dep,
                                      const uint64_t (&msk)[W]) {
  const size_t r = (size_t)(rq.off + node);
  a.depth[r] = dep;
#pragma unroll
  for (int w = 0; w < W; ++w)
    if (w < a.words) a.anc_mask[r * a.words + w] = msk[w];
}

template <int KIND, int W, int NH>
__global__ __launch_bounds__(kThreads) void topology_kernel(TopoArgs a) {
  __shared__ int s_jmp[kThreads];
  __shared__ float s_acc[kThreads];
  __shared__ int s_cnt[kThreads];
  __shared__ uint64_t s_msk[W * kThreads];
  const int tid = threadIdx.x;
  Request rq;
  if (!load_request(a.node_offsets, blockIdx.x, a.max_nodes, a.dev_err, rq)) return;
  const int T = rq.T;
  if (T == 0) return;
  if constexpr (KIND == kTopoJump1) {
    if (tid >= 64) return;   // one wavefront; the others take no part
    int par[W];
    float x[W], cl[W];
    uint64_t msk[W][W];
#pragma unroll
    for (int e = 0; e < W; ++e) {   // lanes past the tree read its last node, as the kernel does
      par[e] = a.parent[rq.off + min(tid + 64 * e, T - 1)];
      x[e] = 0.f;
    }
    if (!wave_topology_jump<W, W>(par, x, T, s_jmp, s_acc, s_msk, cl, msk)) {
      if (tid == 0) report(a.dev_err, TL_EBADTREE);
      return;
    }
#pragma unroll
    for (int e = 0; e < W; ++e) {
      if (tid + 64 * e < T) {
        int c = 0;
#pragma unroll
        for (int w = 0; w < W; ++w) c += __popcll(msk[e][w]);
        store_topology<W>(a, rq, tid + 64 * e, c - 1, msk[e]);
      }
    }
    return;
  }
  const bool wave_path = KIND == kTopoWaveN || (KIND == kTopoGdn && T <= 64);
  if (wave_path) {
    if (tid >= 64) return;   // one wavefront; the others take no part
    // lanes >= T read node 0, as the verify kernels do (ignored by the routine)
    const int par = a.parent[rq.off + (tid < T ? tid : 0)];
    uint64_t m1 = 0ull;
    int dep = 0;
    bool ok;
    if constexpr (KIND == kTopoWaveN) {
      float x[NH], cl[NH];
#pragma unroll
      for (int hh = 0; hh < NH; ++hh) x[hh] = 0.f;
      ok = wave_topology_n<NH>(par, T, x, cl, m1);
      dep = __popcll(m1) - 1;
    } else {
      float cl;
      ok = wave_topology(par, T, 0.f, dep, cl, m1);
    }
    if (!ok) {
      if (tid == 0) report(a.dev_err, TL_EBADTREE);
      return;
    }
    if (tid < T) {
      uint64_t msk[W];
#pragma unroll
      for (int w = 0; w < W; ++w) msk[w] = w == 0 ? m1 : 0ull;
      store_topology<W>(a, rq, tid, dep, msk);
    }
    return;
  }
  int dep;
  float cl;
  uint64_t msk[W];
  const int par = (tid < T) ? a.parent[rq.off + tid] : -1;
  if (!build_topology<W, true>(par, T, 0.f, s_jmp, s_acc, s_cnt, s_msk, dep, cl, msk)) {
    if (tid == 0) report(a.dev_err, TL_EBADTREE);
    return;
  }
  if (tid < T) store_topology<W>(a, rq, tid, dep, msk);
}

template <int KIND, int W, int NH = 1>
static tl_status launch_topo(const TopoArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL((topology_kernel<KIND, W, NH>), dim3((unsigned)a.batch), dim3(kThreads), 0,
                     stream, a);
  return hipGetLastError() == hipSuccess ? TL_OK : TL_EHIP;
}

tl_status launch_topology(const tl_problem& p, const TopoArgs& a, hipStream_t stream) {
  if (a.batch == 0) return TL_OK;
  const int tm = (p.max_nodes + 15) & ~15;
  const int W = tm > 128 ? 4 : (tm > 64 ? 2 : 1);
  const bool mfma = p.in_dtype == TL_BF16 && p.d_k >= 32;
  if (mfma && p.mode == TL_MODE_GDN && p.d_k == 128 && tm <= 128)
    return W == 1 ? launch_topo<kTopoJump1, 1>(a, stream) : launch_topo<kTopoJump1, 2>(a, stream);
  if (mfma && p.mode == TL_MODE_GLA && tm > 64)
    return W == 2 ? launch_topo<kTopoJump1, 2>(a, stream) : launch_topo<kTopoJump1, 4>(a, stream);
  if (mfma && p.mode == TL_MODE_GLA && tm <= 64)
    return (p.num_v_heads / p.num_qk_heads) % 2 == 0 ? launch_topo<kTopoWaveN, 1, 2>(a, stream)
                                                     : launch_topo<kTopoWaveN, 1, 1>(a, stream);
  if (mfma && p.mode == TL_MODE_GDN && verify_tiled_lds_bytes(p.d_k, tm, W) > 160 * 1024)
    return launch_topo<kTopoGdn, 4>(a, stream);
  switch (W) {
    case 1: return launch_topo<kTopoLds, 1>(a, stream);
    case 2: return launch_topo<kTopoLds, 2>(a, stream);
    default: return launch_topo<kTopoLds, 4>(a, stream);
  }
}

}  // namespace tl
