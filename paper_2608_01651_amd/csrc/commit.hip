// Accepted-path commit (§4.4, Eq. accepted-commit).
//
// S_new = P_a S_pre + (D_a K_a)^T U_a is, by Lemma 1, the post-update state
// of the terminal node a, i.e. the recurrence replayed along the accepted
// path from S_pre.  The kernel replays it in fp32, in place:
//   gated linear attention:  S <- gamma S + v k^T
//   gated delta rule:        u = beta (v - gamma S k),  S <- gamma S + u k^T
// (stored orientation: S is the slot's [d_v, d_k] matrix).  Rows of the
// stored state evolve independently under both rules, so one workgroup owns a
// whole (request, v-head) slot with no cross-workgroup reduction.  Each
// workgroup reads its whole slot before it writes any of it.  An empty path
// leaves the slot untouched.
#include <hip/hip_runtime.h>

#include "tl_device.h"
#include "tl_kernels.h"

namespace tl {

constexpr int kCommitChunk = 32;   // path steps staged in LDS at a time

template <int MODE, int D, bool F32IN>
__global__ __launch_bounds__(kThreads) void commit_kernel(CommitArgs a) {
  constexpr int LPR = D / 4;                        // lanes per state row (4 floats each)
  constexpr int RPP = kThreads / LPR;               // rows per pass of the block
  constexpr int PASSES = (D + RPP - 1) / RPP;
  constexpr bool GDN = (MODE == TL_MODE_GDN);
  __shared__ __align__(16) float s_k[kCommitChunk * D];
  __shared__ __align__(16) float s_v[kCommitChunk * D];
  __shared__ float s_gam[kCommitChunk];
  __shared__ float s_beta[kCommitChunk];
  __shared__ int s_row[kCommitChunk];

  const int tid = threadIdx.x;
  const int b = blockIdx.x / a.Hv, h = blockIdx.x % a.Hv;
  const int hq = h / (a.Hv / a.Hk);

  Request rq;
  if (!load_request(a.node_offsets, b, a.max_nodes, a.dev_err, rq)) return;
  const int T = rq.T, off = rq.off;
  const int p0 = a.path_offsets[b], p1 = a.path_offsets[b + 1];
  const int Lp = p1 - p0;
  if (p0 < 0 || Lp < 0) {
    if (tid == 0) report(a.dev_err, TL_EINVAL);
    return;
  }
  const int sidx = a.slot ? a.slot[b] : b;
  if (sidx < 0 || sidx >= a.num_slots) {
    if (tid == 0) report(a.dev_err, TL_EINVAL);
    return;
  }
  // the slot is read first (whole tile into registers) so that its latency
  // overlaps the checks below; nothing is written before they pass
  float* Sp = a.state + ((size_t)sidx * a.Hv + h) * D * D;
  const int col = (tid % LPR) * 4;
  f32x4 st[PASSES];
  if (Lp > 0) {
#pragma unroll
    for (int p = 0; p < PASSES; ++p) {
      const int row = p * RPP + tid / LPR;
      if (row < D) st[p] = *reinterpret_cast<const f32x4*>(Sp + (size_t)row * D + col);
    }
  }
  // forest of request b (one node per thread)
  {
    bool bad = false;
    if (tid < T) {
      const int p = a.parent[off + tid];
      bad = !(p == -1 || (p >= 0 && p < tid));
    }
    if (__syncthreads_or(bad)) {
      if (tid == 0) report(a.dev_err, TL_EBADTREE);
      return;
    }
  }
  // path: a root-first chain of request-local nodes
  {
    bool bad = Lp > T || (Lp > 0 && a.path == nullptr);
    if (!bad && tid < Lp) {
      const int node = a.path[p0 + tid];
      const int want = (tid == 0) ? -1 : a.path[p0 + tid - 1];
      bad = !(node >= 0 && node < T) || a.parent[off + node] != want;
    }
    if (__syncthreads_or(bad)) {
      if (tid == 0) report(a.dev_err, TL_EBADPATH);
      return;
    }
  }
  if (Lp == 0) return;

  const size_t qk_row = (size_t)a.Hk * D, v_row = (size_t)a.Hv * D;
  for (int c0 = 0; c0 < Lp; c0 += kCommitChunk) {
    const int n = min(kCommitChunk, Lp - c0);
    __syncthreads();   // previous chunk fully consumed
    if (tid < n) {
      const int r = off + a.path[p0 + c0 + tid];
      s_row[tid] = r;
      s_gam[tid] = __expf(a.g[(size_t)r * a.Hv + h]);
      if constexpr (GDN) s_beta[tid] = a.beta[(size_t)r * a.Hv + h];
    }
    __syncthreads();
    for (int x = tid * 4; x < n * D; x += kThreads * 4) {
      const int t = x / D, e = x % D;
      const int r = s_row[t];
      *reinterpret_cast<f32x4*>(s_k + x) = load4<F32IN>(a.k, (size_t)r * qk_row + (size_t)hq * D + e);
      *reinterpret_cast<f32x4*>(s_v + x) = load4<F32IN>(a.v, (size_t)r * v_row + (size_t)h * D + e);
    }
    __syncthreads();
    for (int t = 0; t < n; ++t) {
      const float gam = s_gam[t];
      const f32x4 kv = *reinterpret_cast<const f32x4*>(s_k + t * D + col);
#pragma unroll
      for (int p = 0; p < PASSES; ++p) {
        const int row = p * RPP + tid / LPR;
        const float vv = s_v[t * D + (row < D ? row : 0)];
        if constexpr (!GDN) {
          st[p] = gam * st[p] + vv * kv;
        } else {
          float part = st[p][0] * kv[0] + st[p][1] * kv[1] + st[p][2] * kv[2] + st[p][3] * kv[3];
#pragma unroll
          for (int o = 1; o < LPR; o <<= 1) part += __shfl_xor(part, o, 64);
          const float u = s_beta[t] * (vv - gam * part);
          st[p] = gam * st[p] + u * kv;
        }
      }
    }
  }
#pragma unroll
  for (int p = 0; p < PASSES; ++p) {
    const int row = p * RPP + tid / LPR;
    if (row < D) *reinterpret_cast<f32x4*>(Sp + (size_t)row * D + col) = st[p];
  }
}

template <int MODE, int D, bool F32IN>
static tl_status launch_one(const CommitArgs& a, hipStream_t stream) {
  const long blocks = (long)a.batch * a.Hv;
  if (blocks == 0) return TL_OK;
  if (blocks > 0x7fffffffL) return TL_EINVAL;
  hipLaunchKernelGGL((commit_kernel<MODE, D, F32IN>), dim3((unsigned)blocks), dim3(kThreads), 0,
                     stream, a);
  return hipGetLastError() == hipSuccess ? TL_OK : TL_EHIP;
}

template <int MODE, bool F32IN>
static tl_status dispatch_d(int d, const CommitArgs& a, hipStream_t stream) {
  switch (d) {
    case 16: return launch_one<MODE, 16, F32IN>(a, stream);
    case 32: return launch_one<MODE, 32, F32IN>(a, stream);
    case 64: return launch_one<MODE, 64, F32IN>(a, stream);
    case 128: return launch_one<MODE, 128, F32IN>(a, stream);
    default: return TL_EUNSUPPORTED;
  }
}

tl_status launch_commit(const tl_problem& p, const CommitArgs& a, hipStream_t stream) {
  if (p.mode == TL_MODE_GLA)
    return p.in_dtype == TL_F32 ? dispatch_d<TL_MODE_GLA, true>(p.d_k, a, stream)
                                : dispatch_d<TL_MODE_GLA, false>(p.d_k, a, stream);
  return p.in_dtype == TL_F32 ? dispatch_d<TL_MODE_GDN, true>(p.d_k, a, stream)
                              : dispatch_d<TL_MODE_GDN, false>(p.d_k, a, stream);
}

}  // namespace tl
