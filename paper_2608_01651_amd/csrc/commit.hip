// Accepted-path commit (§4.4, Eq. accepted-commit).
//
// S_new = P_a S_pre + (D_a K_a)^T U_a is, by Lemma 1, the post-update state
// of the terminal node a, i.e. the recurrence replayed along the accepted
// path from S_pre.  The kernel replays it in fp32, in place:
//   gated linear attention:  S <- gamma S + v k^T
//   gated delta rule:        u = beta (v - gamma S k),  S <- gamma S + u k^T
// (stored orientation: S is the slot's [d_v, d_k] matrix).  Rows of the
// stored state evolve independently under both rules (the delta rule's
// S k is a per-row dot product), so each block of rows is replayed on its
// own, and nothing crosses workgroups.  A workgroup checks the forest and the
// path before it writes anything, and every block is read before it is
// written; an empty path leaves the slot untouched.  The state is read and
// written once, with non-temporal loads and stores.
#include <hip/hip_runtime.h>

#include "tl_device.h"
#include "tl_kernels.h"

namespace tl {

constexpr int kCommitChunk = 32;   // path steps staged in LDS at a time

template <int D>
struct CommitShape {
  static constexpr int ROWS = (D >= 64) ? 32 : D;   // state rows per streamed block
  static constexpr int NRB = D / ROWS;              // blocks per (request, v-head) slot
  static constexpr int LPR = D / 4;                 // lanes per row (4 floats each)
  static constexpr int RPP = kThreads / LPR;        // rows per pass of the workgroup
  static constexpr int PASSES = (ROWS + RPP - 1) / RPP;
};

// One workgroup per (request, v-head) slot.  The path is validated and its
// rows (k, v, gates) are staged in LDS once; the slot is then replayed and
// stored in blocks of ROWS rows, whose loads are all issued at the start
// (delta rule: two blocks at a time).
template <int MODE, int D, bool F32IN>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4))) void commit_kernel(CommitArgs a) {
  using SH = CommitShape<D>;
  constexpr int ROWS = SH::ROWS, NRB = SH::NRB, LPR = SH::LPR, RPP = SH::RPP, PASSES = SH::PASSES;
  constexpr bool GDN = (MODE == TL_MODE_GDN);
  __shared__ __align__(16) float s_k[kCommitChunk * D];
  __shared__ __align__(16) float s_v[kCommitChunk * D];
  __shared__ float s_gam[kCommitChunk];
  __shared__ float s_beta[kCommitChunk];
  __shared__ int s_row[kCommitChunk];
  __shared__ int s_par[kMaxNodes];

  const int tid = threadIdx.x;
  TL_TRACE_POINT(a, 0);
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
  TL_TRACE_POINT(a, 1);

  // state blocks are read first so that their latency overlaps the checks
  // below; nothing is written before they pass
  float* Sp = a.state + ((size_t)sidx * a.Hv + h) * D * D;
  const int col = (tid % LPR) * 4;
  const int rsub = tid / LPR;
  auto load_block = [&](int rb, f32x4 (&st)[PASSES]) {
#pragma unroll
    for (int p = 0; p < PASSES; ++p) {
      const int row = p * RPP + rsub;
      if (row < ROWS)
        st[p] = __builtin_nontemporal_load(
            reinterpret_cast<const f32x4*>(Sp + (size_t)(rb * ROWS + row) * D + col));
    }
  };
  auto store_block = [&](int rb, const f32x4 (&st)[PASSES]) {
#pragma unroll
    for (int p = 0; p < PASSES; ++p) {
      const int row = p * RPP + rsub;
      if (row < ROWS)
        __builtin_nontemporal_store(st[p], reinterpret_cast<f32x4*>(Sp + (size_t)(rb * ROWS + row) * D + col));
    }
  };
  // gated linear attention keeps every block of the slot in registers (all
  // loads in flight at once); the delta rule needs more registers for its
  // row reductions and streams the blocks through two buffers
  constexpr int NBUF = GDN ? (NRB < 2 ? NRB : 2) : NRB;
  f32x4 sb[NBUF][PASSES];
  if (Lp > 0) {
#pragma unroll
    for (int rb = 0; rb < NBUF; ++rb) load_block(rb, sb[rb]);
  }

  // forest of request b (one node per thread) and the path, loaded together;
  // the path's links are then checked against the parents in LDS
  int par = -1, node = -1;
  if (tid < T) par = a.parent[off + tid];
  const bool path_ok = !(Lp > T || (Lp > 0 && a.path == nullptr));
  if (path_ok && tid < Lp) node = a.path[p0 + tid];
  if (tid < T) s_par[tid] = par;
  const bool bad_tree = (tid < T) && !(par == -1 || (par >= 0 && par < tid));
  const bool node_in = node >= 0 && node < T;
  TL_TRACE_POINT(a, 2);
  if (__syncthreads_or(bad_tree)) {
    if (tid == 0) report(a.dev_err, TL_EBADTREE);
    return;
  }
  {
    bool bad = !path_ok;
    if (!bad && tid < Lp) {
      const int want = (tid == 0) ? -1 : a.path[p0 + tid - 1];
      bad = !node_in || s_par[node] != want;
    }
    if (__syncthreads_or(bad)) {
      if (tid == 0) report(a.dev_err, TL_EBADPATH);
      return;
    }
  }
  if (Lp == 0) return;
  TL_TRACE_POINT(a, 3);

  const size_t qk_row = (size_t)a.Hk * D, v_row = (size_t)a.Hv * D;
  // stage path steps [c0, c0 + n): row ids and gates, then k and v rows
  auto stage = [&](int c0, int n) {
    if (tid < n) {
      const int r = off + a.path[p0 + c0 + tid];
      s_row[tid] = r;
      s_gam[tid] = __expf(a.g[(size_t)r * a.Hv + h]);
      if constexpr (GDN) s_beta[tid] = a.beta[(size_t)r * a.Hv + h];
    }
    __syncthreads();
    for (int x = tid * 4; x < n * D; x += kThreads * 4) {
      const int t = x / D, e = x % D;
      const size_t r = (size_t)s_row[t];
      *reinterpret_cast<f32x4*>(s_k + x) = load4<F32IN>(a.k, r * qk_row + (size_t)hq * D + e);
      *reinterpret_cast<f32x4*>(s_v + x) = load4<F32IN>(a.v, r * v_row + (size_t)h * D + e);
    }
    __syncthreads();
  };
  // replay staged steps [0, n) on the rows of block rb
  auto replay = [&](int rb, int n, f32x4 (&st)[PASSES]) {
    for (int t = 0; t < n; ++t) {
      const float gam = s_gam[t];
      const f32x4 kv = *reinterpret_cast<const f32x4*>(s_k + t * D + col);
#pragma unroll
      for (int p = 0; p < PASSES; ++p) {
        const int row = p * RPP + rsub;
        const float vv = s_v[t * D + rb * ROWS + (row < ROWS ? row : 0)];
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
  };

  if (Lp <= kCommitChunk) {
    stage(0, Lp);
    TL_TRACE_POINT(a, 4);
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) {
      replay(rb, Lp, sb[rb % NBUF]);
      store_block(rb, sb[rb % NBUF]);
      if (rb + NBUF < NRB) load_block(rb + NBUF, sb[rb % NBUF]);
    }
  } else {
    // long paths: the steps are staged chunk by chunk for every block
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) {
      for (int c0 = 0; c0 < Lp; c0 += kCommitChunk) {
        const int n = min(kCommitChunk, Lp - c0);
        __syncthreads();   // the previous chunk is fully consumed
        stage(c0, n);
        replay(rb, n, sb[rb % NBUF]);
      }
      store_block(rb, sb[rb % NBUF]);
      if (rb + NBUF < NRB) load_block(rb + NBUF, sb[rb % NBUF]);
    }
  }
  TL_TRACE_POINT(a, 5);
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
