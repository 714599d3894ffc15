// Tree-parallel verification (Theorem 1, §4.1; value tiling of §4.2).
//
// One workgroup handles one (request b, v-head h, value slice of BV columns).
// For every node i of the request it produces
//   o_i = q_scale * ( P_i * S_pre^T q_i  +  sum_{j in Anc(i) u {i}} c_ij u_j )
// with P_i = exp(cl_i) the decay product along the root path (cl = cumulative
// log-decay), c_ij = exp(cl_i - cl_j) (q_i . k_j) and
//   u_j = v_j                                   (gated linear attention), or
//   u   = (I + G)^{-1} beta (v - P K S_pre)     (gated delta rule, Lemma 2),
//         G_ij = beta_i exp(cl_i - cl_j) (k_i . k_j) for strict ancestors j.
// No per-node state is formed; S_pre is read once, and only O leaves the chip.
//
// MFMA path (bf16 inputs, d >= 32, trees of 16 nodes or more):
//  1. the request's parents and gates are loaded first, then the state slice
//     goes straight into MFMA A-operand registers (rows = value channels of
//     the stored [d_v, d_k] slot), and K (plus the value slice for GLA) is
//     copied global -> LDS without touching registers;
//  2. pointer jumping over the parents gives every node its M+ row (64-bit
//     words), and the cumulative log-decay, while those loads are in flight;
//     the fp32 state is then split into bf16 hi + lo so the bf16 MFMA keeps
//     ~2^-17 relative accuracy;
//  3. nodes are processed in tiles of 16 (topological order, so every ancestor
//     of a tile lies in the same or an earlier tile):
//       a. B0 = S Q^T (and S K^T for the delta rule) on MFMA;
//       b. K Q^T (and K K^T) tiles against every tile holding an ancestor of
//          the tile, on MFMA; only ancestor entries are kept, indexed by the
//          ancestor's depth (a node has exactly one ancestor per depth);
//       c. delta rule: R = beta (V - P (K S^T)), then forward substitution
//          along the tree (earlier tiles are final; inside the tile, level by
//          level), U kept in LDS;
//       d. readout O = P B0 + sum over the root path of c_ij u_j, fp32 out.
//     Ancestors are enumerated from the node's M+ bits in index order, which
//     is root-first, so the k-th set bit is the ancestor at depth k.
// Vector path (fp32 inputs, d = 16, trees of fewer than 16 nodes): the same
// steps with vector ALU products.
//
// Files: verify_gla_small.h (gated linear attention on MFMA, trees of <= 64
// nodes), verify_gla_large.hip (its own kernel: gated linear attention over
// trees of 65..256 nodes), verify_gdn_dense.hip (its own kernel: the delta
// rule at d = 128 over node caps of up to 128), verify_tiled.hip (its own
// kernel: the delta rule node tile by node tile, where that layout fits in
// LDS), verify_gdn.h (the delta rule's per-wave MFMA path, for shapes whose
// tile-by-tile layout does not fit in LDS), verify_vector.h (vector path),
// verify_common.h (layouts).
#include <hip/hip_runtime.h>

#include "tl_device.h"
#include "tl_kernels.h"
#include "verify_common.h"
#include "verify_gdn.h"
#include "verify_gla_small.h"
#include "verify_vector.h"

namespace tl {

template <int MODE, int D, int BV, bool F32IN, int W, int NH>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(NH == 2 ? 2 : 1))) void verify_kernel(VerifyArgs a) {
  constexpr int NSL = D / BV;              // value slices per head
  constexpr bool CAN_MFMA = !F32IN && D >= 32;
  const int tid = threadIdx.x;
  lds_poison(a.lds_bytes);
  TL_TRACE_POINT(a, 0);

  // ---- block -> (request, qk-head, first v-head, slice).  A block serves NH
  // v-heads of one qk-head.  Consecutive block ids go to different XCDs
  // (round robin over 8); all blocks that read the same request's q/k rows
  // are given ids 8 apart so they share one XCD's L2.
  const int grp = a.Hv / a.Hk;
  const int GS = (grp / NH) * NSL;
  const int nshare = a.batch * a.Hk;
  const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
  const int sh = (local / GS) * 8 + xcd;
  if (sh >= nshare) return;
  const int w_in = local % GS;
  Unit u;
  u.b = sh / a.Hk;
  u.hq = sh % a.Hk;
  u.h = u.hq * grp + (w_in / NSL) * NH;
  u.slice = w_in % NSL;
  u.tm = a.tm;

  // the slot is read with the node range (independent loads, one round trip)
  u.sidx = a.slot ? a.slot[u.b] : u.b;
  Request rq;
  if (!load_request(a.node_offsets, u.b, a.max_nodes, a.dev_err, rq)) return;
  u.off = rq.off;
  u.T = rq.T;
  if (u.T == 0) return;
  if (u.sidx < 0 || u.sidx >= a.num_slots) {
    if (tid == 0) report(a.dev_err, TL_EINVAL);
    return;
  }
  if constexpr (CAN_MFMA) {
    if (u.T >= kTile) {
      if constexpr (MODE == TL_MODE_GLA) {
        static_assert(W == 1, "larger trees of gated linear attention run in the large-tree kernel");
        verify_gla_small<D, BV, NH>(a, u);
      } else {
        verify_gdn_mfma<MODE, D, BV, W>(a, u);
      }
      TL_TRACE_POINT(a, 15);
      return;
    }
  }
#pragma unroll
  for (int hh = 0; hh < NH; ++hh) {
    if (hh) __syncthreads();   // the previous head is done with the LDS
    Unit uh = u;
    uh.h = u.h + hh;
    verify_vector<MODE, D, BV, F32IN, W>(a, uh);
  }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
template <int MODE, int D, int BV, bool F32IN, int W, int NH>
static tl_status launch_one(const VerifyArgs& a, hipStream_t stream) {
  constexpr int NSL = D / BV;
  constexpr bool CAN_MFMA = !F32IN && D >= 32;
  // a block may take the vector path or (at least 16 nodes) the MFMA path
  VerifyLayout L = verify_layout(MODE, D, BV, F32IN ? 4 : 2, a.tm, W, false);
  if (CAN_MFMA) {
    int t;
    if (MODE == TL_MODE_GLA) t = gla_small_layout(D, BV, NH).total;
    else t = verify_layout(MODE, D, BV, 2, a.tm, W, true).total;
    if (t > L.total) L.total = t;
  }
  const int grp = a.Hv / a.Hk;
  const long nshare = (long)a.batch * a.Hk;
  const long blocks = 8 * ((nshare + 7) / 8) * (grp / NH) * NSL;
  if (blocks == 0) return TL_OK;
  if (blocks > 0x7fffffffL) return TL_EINVAL;
  auto kern = verify_kernel<MODE, D, BV, F32IN, W, NH>;
  if (L.total > 160 * 1024) return TL_EUNSUPPORTED;
  if (L.total > 64 * 1024) {
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                            hipFuncAttributeMaxDynamicSharedMemorySize, L.total) != hipSuccess)
      return TL_EHIP;
  }
  VerifyArgs b = a;
  b.lds_bytes = L.total;
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kThreads), L.total, stream, b);
  return hipGetLastError() == hipSuccess ? TL_OK : TL_EHIP;
}

// W = 64-bit words per ancestor mask (trees of <= 64, 128, 256 nodes).  The
// delta rule with d = 128 keeps U [tm][BV] in LDS, so 256-node trees use
// 32-column value slices to stay within the 160 KB of LDS.  Gated linear
// attention over trees of <= 64 nodes serves two grouped v-heads per block
// when the group size is even (bf16 inputs, d >= 32).
template <int MODE, int D, int BV, bool F32IN>
static tl_status dispatch_w(const VerifyArgs& a, hipStream_t stream) {
  if constexpr (F32IN) {
    return launch_one<MODE, D, BV, F32IN, 4, 1>(a, stream);
  } else if constexpr (MODE == TL_MODE_GLA && D >= 32) {
    // trees of more than 64 nodes are served by the large-tree kernel
    if (a.tm > 64) return TL_EUNSUPPORTED;
    if ((a.Hv / a.Hk) % 2 == 0) return launch_one<MODE, D, BV, F32IN, 1, 2>(a, stream);
    return launch_one<MODE, D, BV, F32IN, 1, 1>(a, stream);
  } else {
    if (a.tm > 128) {
      if constexpr (MODE == TL_MODE_GDN && D == 128) return launch_one<MODE, D, 32, F32IN, 4, 1>(a, stream);
      return launch_one<MODE, D, BV, F32IN, 4, 1>(a, stream);
    }
    if (a.tm > 64) return launch_one<MODE, D, BV, F32IN, 2, 1>(a, stream);
    return launch_one<MODE, D, BV, F32IN, 1, 1>(a, stream);
  }
}

template <int MODE, bool F32IN>
static tl_status dispatch_d(int d, const VerifyArgs& a, hipStream_t stream) {
  switch (d) {
    case 16: return dispatch_w<MODE, 16, 16, F32IN>(a, stream);
    case 32: return dispatch_w<MODE, 32, 32, F32IN>(a, stream);
    case 64: return dispatch_w<MODE, 64, 64, F32IN>(a, stream);
    case 128: return dispatch_w<MODE, 128, (MODE == TL_MODE_GDN ? 64 : 128), F32IN>(a, stream);
    default: return TL_EUNSUPPORTED;
  }
}

tl_status launch_verify(const tl_problem& p, const VerifyArgs& a, hipStream_t stream) {
  // the delta rule at d = 128 over node caps of up to 128: the correction
  // system inverted once per workgroup (verify_gdn_dense.hip)
  if (p.mode == TL_MODE_GDN && p.in_dtype == TL_BF16 && p.d_k == 128 && a.tm <= 128)
    return launch_verify_gdn_dense(p, a, stream);
  // bf16 inputs, d >= 32: gated linear attention over trees of more than 64
  // nodes, node tile by node tile with every operand resident on chip
  // (verify_gla_large.hip); the delta rule wherever its tile-sequential
  // layout fits in LDS (node caps of up to 160 at d = 128, verify_tiled.hip)
  if (p.in_dtype == TL_BF16 && p.d_k >= 32) {
    if (p.mode == TL_MODE_GLA && a.tm > 64) return launch_verify_gla_large(p, a, stream);
    const int W = a.tm > 128 ? 4 : (a.tm > 64 ? 2 : 1);
    if (p.mode == TL_MODE_GDN && verify_tiled_lds_bytes(p.d_k, a.tm, W) <= 160 * 1024)
      return launch_verify_tiled(p, a, stream);
  }
  if (p.mode == TL_MODE_GLA)
    return p.in_dtype == TL_F32 ? dispatch_d<TL_MODE_GLA, true>(p.d_k, a, stream)
                                : dispatch_d<TL_MODE_GLA, false>(p.d_k, a, stream);
  return p.in_dtype == TL_F32 ? dispatch_d<TL_MODE_GDN, true>(p.d_k, a, stream)
                              : dispatch_d<TL_MODE_GDN, false>(p.d_k, a, stream);
}

}  // namespace tl
