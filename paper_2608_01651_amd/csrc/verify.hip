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
// Work per workgroup:
//  1. issue the loads of the state slice straight into MFMA A-operand
//     registers (rows of the stored [d_v, d_k] slot), then split each fp32
//     element into bf16 hi + lo so the bf16 MFMA keeps ~2^-17 relative accuracy;
//  2. build the tree topology by pointer jumping (depth, M+ rows as 64-bit
//     words, cumulative log-decay) in LDS, and stage the value slice (GLA);
//  3. walk the nodes in tiles of 16 (topological order, so every ancestor of a
//     tile lies in the same or an earlier tile):
//       a. B0 = S Q^T (and S K^T for the delta rule) for the tile on MFMA;
//       b. Q K^T (and K K^T) tiles against every earlier tile that holds an
//          ancestor of the tile, on MFMA; only the ancestor entries are kept,
//          as coefficients indexed by the ancestor's depth (a node has exactly
//          one ancestor per depth);
//       c. delta rule: R = beta (V - P (K S^T)), then forward substitution
//          along the tree (earlier tiles are final; inside the tile, level by
//          level), U kept in LDS;
//       d. readout O = P B0 + sum over the root path of c_ij u_j, stored as fp32.
//  Trees with fewer than 16 nodes (and fp32 inputs, and d_k = 16) take the
//  same steps with vector ALU products instead of MFMA.
#include <hip/hip_runtime.h>

#include "tl_device.h"
#include "tl_kernels.h"

namespace tl {

// ---------------------------------------------------------------------------
// LDS layout (bytes); identical on host and device.
// ---------------------------------------------------------------------------
struct VerifyLayout {
  int par, depth, cl, beta, mask, tmask, uni, vbuf, total;
};

__host__ __device__ inline int align16(int x) { return (x + 15) & ~15; }

__host__ __device__ inline VerifyLayout verify_layout(int mode, int BV, int vbytes, int tm) {
  VerifyLayout L;
  int o = 0;
  L.par = o;   o += align16(tm * 4);
  L.depth = o; o += align16(tm * 4);
  L.cl = o;    o += align16(tm * 4);
  L.beta = o;  o += (mode == TL_MODE_GDN) ? align16(tm * 4) : 0;
  L.mask = o;  o += tm * 4 * 8;
  L.tmask = o; o += (tm / kTile) * 4 * 8;
  L.uni = o;
  // union: topology scratch | per-tile coefficients (c, and G for the delta rule)
  int topo = kThreads * (4 + 4 + 4) + kThreads * 4 * 8;
  int coef = kTile * tm * 4 * ((mode == TL_MODE_GDN) ? 2 : 1);
  o += align16(topo > coef ? topo : coef);
  L.vbuf = o;  // GLA: staged values [tm][BV] (input dtype); GDN: U [tm][BV] fp32
  o += (mode == TL_MODE_GDN) ? tm * BV * 4 : tm * BV * vbytes;
  L.total = o;
  return L;
}

template <int MODE, int D, int BV, bool F32IN>
__global__ __launch_bounds__(kThreads) void verify_kernel(VerifyArgs a) {
  constexpr int NSL = D / BV;              // value slices per head
  constexpr int KS = D / 32;               // 32-wide K chunks of the MFMA
  constexpr int MTILES = BV / kTile;       // 16-row value tiles in the slice
  constexpr int MT = (MTILES + kWaves - 1) / kWaves;  // tiles per wave
  constexpr bool CAN_MFMA = !F32IN && D >= 32;
  constexpr bool GDN = (MODE == TL_MODE_GDN);
  using VT = typename std::conditional<F32IN, float, __bf16>::type;
  extern __shared__ __align__(16) unsigned char lds[];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, lr = lane & 15, lg = lane >> 4;

  // ---- block -> (request, qk-head, v-head, slice).  Consecutive block ids go
  // to different XCDs (round robin over 8); all blocks that read the same
  // request's q/k rows are given ids 8 apart so they share one XCD's L2.
  const int grp = a.Hv / a.Hk;
  const int GS = grp * NSL;
  const int nshare = a.batch * a.Hk;
  const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
  const int sh = (local / GS) * 8 + xcd;
  if (sh >= nshare) return;
  const int w_in = local % GS;
  const int b = sh / a.Hk, hq = sh % a.Hk;
  const int h = hq * grp + w_in / NSL;
  const int slice = w_in % NSL;

  Request rq;
  if (!load_request(a.node_offsets, b, a.max_nodes, a.dev_err, rq)) return;
  const int T = rq.T, off = rq.off;
  if (T == 0) return;
  const int sidx = a.slot ? a.slot[b] : b;
  if (sidx < 0 || sidx >= a.num_slots) {
    if (tid == 0) report(a.dev_err, TL_EINVAL);
    return;
  }
  const bool use_mfma = CAN_MFMA && T >= kTile;
  const int tm = a.tm;
  const VerifyLayout L = verify_layout(MODE, BV, (int)sizeof(VT), tm);
  int* s_par = reinterpret_cast<int*>(lds + L.par);
  int* s_depth = reinterpret_cast<int*>(lds + L.depth);
  float* s_cl = reinterpret_cast<float*>(lds + L.cl);
  float* s_beta = reinterpret_cast<float*>(lds + L.beta);
  uint64_t* s_mask = reinterpret_cast<uint64_t*>(lds + L.mask);
  uint64_t* s_tmask = reinterpret_cast<uint64_t*>(lds + L.tmask);
  float* s_c = reinterpret_cast<float*>(lds + L.uni);
  float* s_G = s_c + kTile * tm;
  VT* s_v = reinterpret_cast<VT*>(lds + L.vbuf);
  float* s_u = reinterpret_cast<float*>(lds + L.vbuf);

  const float* Sp = a.state + ((size_t)sidx * a.Hv + h) * D * D;
  const size_t qk_row = (size_t)a.Hk * D;   // elements between consecutive nodes
  const size_t v_row = (size_t)a.Hv * D;

  // ---- 1. state slice -> registers (A operand rows = value channels)
  f32x4 sraw[MT][KS > 0 ? KS : 1][2];
  if constexpr (CAN_MFMA) {
    if (use_mfma) {
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        const int mt = wave + kWaves * m;
        if (mt < MTILES) {
          const float* row = Sp + (size_t)(slice * BV + kTile * mt + lr) * D;
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            sraw[m][ks][0] = *reinterpret_cast<const f32x4*>(row + ks * 32 + 4 * lg);
            sraw[m][ks][1] = *reinterpret_cast<const f32x4*>(row + ks * 32 + 16 + 4 * lg);
          }
        }
      }
    }
  }

  // ---- 2. topology and cumulative log-decay of v-head h
  for (int x = tid; x < (tm / kTile) * 4; x += kThreads) s_tmask[x] = 0;
  {
    const float gx = (tid < T) ? a.g[(size_t)(off + tid) * a.Hv + h] : 0.f;
    int par, dep;
    float cl;
    uint64_t msk[4];
    int* s_jmp = reinterpret_cast<int*>(lds + L.uni);
    float* s_acc = reinterpret_cast<float*>(s_jmp + kThreads);
    int* s_cnt = reinterpret_cast<int*>(s_acc + kThreads);
    uint64_t* s_msk = reinterpret_cast<uint64_t*>(s_cnt + kThreads);
    if (!build_topology<4, true>(a.parent + off, T, gx, s_jmp, s_acc, s_cnt, s_msk,
                                 par, dep, cl, msk)) {
      if (tid == 0) report(a.dev_err, TL_EBADTREE);
      return;
    }
    __syncthreads();   // topology scratch is dead from here
    if (tid < T) {
      s_par[tid] = par;
      s_depth[tid] = dep;
      s_cl[tid] = cl;
      if constexpr (GDN) s_beta[tid] = a.beta[(size_t)(off + tid) * a.Hv + h];
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        s_mask[tid * 4 + w] = msk[w];
        if (msk[w]) atomicOr(reinterpret_cast<unsigned long long*>(&s_tmask[(tid / kTile) * 4 + w]),
                             (unsigned long long)msk[w]);
      }
    }
  }
  if constexpr (!GDN) {
    // stage the value slice: 16-byte chunks, rows of BV values
    constexpr int CH = 16 / (int)sizeof(VT);
    constexpr int CPR = BV / CH;
    const VT* vsrc = reinterpret_cast<const VT*>(a.v);
    for (int x = tid; x < T * CPR; x += kThreads) {
      const int r = x / CPR, c = x % CPR;
      *reinterpret_cast<f32x4*>(s_v + r * BV + c * CH) =
          *reinterpret_cast<const f32x4*>(vsrc + (size_t)(off + r) * v_row + (size_t)h * D + slice * BV + c * CH);
    }
  }
  __syncthreads();

  // ---- split the state into bf16 hi/lo operands
  bf16x8 shi[MT][KS > 0 ? KS : 1], slo[MT][KS > 0 ? KS : 1];
  if constexpr (CAN_MFMA) {
    if (use_mfma) {
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float x = (e < 4) ? sraw[m][ks][0][e] : sraw[m][ks][1][e - 4];
            __bf16 hi, lo;
            split_bf16(x, hi, lo);
            shi[m][ks][e] = hi;
            slo[m][ks][e] = lo;
          }
    }
  }

  const __bf16* Qb = reinterpret_cast<const __bf16*>(a.q);
  const __bf16* Kb = reinterpret_cast<const __bf16*>(a.k);

  // ---- 3. node tiles
  for (int n0 = 0; n0 < T; n0 += kTile) {
    const int I = n0 / kTile;
    const int i = n0 + lr;            // this lane's node: column of every tile
    const bool iv = i < T;
    const int il = lr;
    const float cli = iv ? s_cl[i] : 0.f;
    const int di = iv ? s_depth[i] : 0;
    const float bi = (GDN && iv) ? s_beta[i] : 0.f;
    f32x4 acc[MT], acck[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
      acck[m] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    if constexpr (CAN_MFMA) {
      if (use_mfma) {
        // a. B0^T = S Q^T (rows: value channels, columns: nodes), K S^T likewise
        bf16x8 qf[KS], kf[KS];
        const __bf16* qrow = Qb + (size_t)(off + i) * qk_row + (size_t)hq * D;
        const __bf16* krow = Kb + (size_t)(off + i) * qk_row + (size_t)hq * D;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          qf[ks] = frag_bf16(qrow, ks, lg, iv);
          if constexpr (GDN) kf[ks] = frag_bf16(krow, ks, lg, iv);
        }
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          if (wave + kWaves * m < MTILES) {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
              acc[m] = mfma16(shi[m][ks], qf[ks], acc[m]);
              acc[m] = mfma16(slo[m][ks], qf[ks], acc[m]);
              if constexpr (GDN) {
                acck[m] = mfma16(shi[m][ks], kf[ks], acck[m]);
                acck[m] = mfma16(slo[m][ks], kf[ks], acck[m]);
              }
            }
          }
        }
        // b. ancestor coefficients from Q K^T (and K K^T) tiles
        uint64_t tmk[4], mi[4];
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          tmk[w] = s_tmask[I * 4 + w];
          mi[w] = iv ? s_mask[i * 4 + w] : 0ull;
        }
        for (int J = wave; J <= I; J += kWaves) {
          const unsigned bits = (unsigned)((tmk[J >> 2] >> ((J & 3) * 16)) & 0xFFFFull);
          if (!bits) continue;                       // no ancestor of this tile in tile J
          const int jr = J * kTile + lr;
          const bool jok = jr < T;
          const __bf16* kjrow = Kb + (size_t)(off + jr) * qk_row + (size_t)hq * D;
          f32x4 qk = f32x4{0.f, 0.f, 0.f, 0.f}, kk = qk;
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            const bf16x8 kj = frag_bf16(kjrow, ks, lg, jok);
            qk = mfma16(kj, qf[ks], qk);             // rows j, column i: k_j . q_i
            if constexpr (GDN) kk = mfma16(kj, kf[ks], kk);
          }
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int j = J * kTile + 4 * lg + r;
            if (iv && j < T && ((mi[j >> 6] >> (j & 63)) & 1ull)) {
              const float dec = __expf(cli - s_cl[j]);
              const int t = s_depth[j];
              s_c[il * tm + t] = dec * qk[r];
              if constexpr (GDN) {
                if (j != i) s_G[il * tm + t] = bi * dec * kk[r];
              }
            }
          }
        }
      }
    }
    if (!use_mfma) {
      // a'. vector products: B0 (and K S^T) for the lane's (node, value rows)
      if (iv) {
        const size_t qbase = (size_t)(off + i) * qk_row + (size_t)hq * D;
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          const int mt = wave + kWaves * m;
          if (mt >= MTILES) continue;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float* srow = Sp + (size_t)(slice * BV + kTile * mt + 4 * lg + r) * D;
            float sq = 0.f, sk = 0.f;
            for (int c = 0; c < D; c += 4) {
              const f32x4 sv = *reinterpret_cast<const f32x4*>(srow + c);
              const f32x4 qv = load4<F32IN>(a.q, qbase + c);
              sq += sv[0] * qv[0] + sv[1] * qv[1] + sv[2] * qv[2] + sv[3] * qv[3];
              if constexpr (GDN) {
                const f32x4 kv = load4<F32IN>(a.k, qbase + c);
                sk += sv[0] * kv[0] + sv[1] * kv[1] + sv[2] * kv[2] + sv[3] * kv[3];
              }
            }
            acc[m][r] = sq;
            acck[m][r] = sk;
          }
        }
      }
      // b'. ancestor coefficients by direct dot products: thread -> (node, depth class)
      {
        const int vi = n0 + (tid & 15);
        if (vi < T) {
          const int dvi = s_depth[vi];
          const float clv = s_cl[vi];
          const float bv = GDN ? s_beta[vi] : 0.f;
          const size_t ibase = (size_t)(off + vi) * qk_row + (size_t)hq * D;
          for (int t = tid >> 4; t <= dvi; t += kThreads / 16) {
            int j = vi;
            for (int u = dvi; u > t; --u) j = s_par[j];
            const size_t jbase = (size_t)(off + j) * qk_row + (size_t)hq * D;
            float qk = 0.f, kk = 0.f;
            for (int c = 0; c < D; c += 4) {
              const f32x4 kj = load4<F32IN>(a.k, jbase + c);
              const f32x4 qi = load4<F32IN>(a.q, ibase + c);
              qk += kj[0] * qi[0] + kj[1] * qi[1] + kj[2] * qi[2] + kj[3] * qi[3];
              if constexpr (GDN) {
                const f32x4 ki = load4<F32IN>(a.k, ibase + c);
                kk += kj[0] * ki[0] + kj[1] * ki[1] + kj[2] * ki[2] + kj[3] * ki[3];
              }
            }
            const float dec = __expf(clv - s_cl[j]);
            s_c[(tid & 15) * tm + t] = dec * qk;
            if constexpr (GDN) {
              if (t < dvi) s_G[(tid & 15) * tm + t] = bv * dec * kk;
            }
          }
        }
      }
    }
    __syncthreads();   // coefficients of this tile are in LDS

    const float Pi = iv ? __expf(cli) : 0.f;
    float* orow = a.out + (size_t)(off + i) * v_row + (size_t)h * D + slice * BV;

    if constexpr (!GDN) {
      // d. readout: O = P B0 + sum_{j on the root path} c_ij v_j
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        const int mt = wave + kWaves * m;
        if (mt >= MTILES || !iv) continue;
        const int vl = kTile * mt + 4 * lg;
        f32x4 o = Pi * acc[m];
        int j = i, t = di;
        while (j >= 0) {
          const float c = s_c[il * tm + t];
          const VT* vp = s_v + j * BV + vl;
          o += c * f32x4{(float)vp[0], (float)vp[1], (float)vp[2], (float)vp[3]};
          j = s_par[j];
          --t;
        }
        *reinterpret_cast<f32x4*>(orow + vl) = a.q_scale * o;
      }
    } else {
      // c. R = beta (V - P (K S^T)), minus the contributions of ancestors in
      //    earlier tiles (their u rows are final)
      f32x4 rr[MT];
      int mylev = -1;
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        const int mt = wave + kWaves * m;
        rr[m] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (mt >= MTILES || !iv) continue;
        const int vl = kTile * mt + 4 * lg;
        const f32x4 vv = load4<F32IN>(a.v, (size_t)(off + i) * v_row + (size_t)h * D + slice * BV + vl);
        rr[m] = bi * (vv - Pi * acck[m]);
        int j = s_par[i], t = di - 1;
        while (j >= n0) { j = s_par[j]; --t; }
        while (j >= 0) {
          const float gij = s_G[il * tm + t];
          rr[m] -= gij * *reinterpret_cast<const f32x4*>(s_u + j * BV + vl);
          j = s_par[j];
          --t;
        }
      }
      if (iv) {   // in-tile level = number of strict ancestors inside this tile
        mylev = 0;
        for (int j = s_par[i]; j >= n0; j = s_par[j]) ++mylev;
      }
      //    forward substitution inside the tile, one level at a time
      for (int lev = 0; __syncthreads_or(mylev >= lev); ++lev) {
        if (mylev == lev) {
#pragma unroll
          for (int m = 0; m < MT; ++m) {
            const int mt = wave + kWaves * m;
            if (mt >= MTILES) continue;
            const int vl = kTile * mt + 4 * lg;
            int j = s_par[i], t = di - 1;
            while (j >= n0) {
              rr[m] -= s_G[il * tm + t] * *reinterpret_cast<const f32x4*>(s_u + j * BV + vl);
              j = s_par[j];
              --t;
            }
            *reinterpret_cast<f32x4*>(s_u + i * BV + vl) = rr[m];
          }
        }
      }
      // d. readout: O = P B0 + sum_{j on the root path} c_ij u_j
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        const int mt = wave + kWaves * m;
        if (mt >= MTILES || !iv) continue;
        const int vl = kTile * mt + 4 * lg;
        f32x4 o = Pi * acc[m];
        int j = i, t = di;
        while (j >= 0) {
          o += s_c[il * tm + t] * *reinterpret_cast<const f32x4*>(s_u + j * BV + vl);
          j = s_par[j];
          --t;
        }
        *reinterpret_cast<f32x4*>(orow + vl) = a.q_scale * o;
      }
    }
    __syncthreads();   // the next tile rewrites the coefficients
  }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
template <int MODE, int D, int BV, bool F32IN>
static tl_status launch_one(const VerifyArgs& a, hipStream_t stream) {
  constexpr int NSL = D / BV;
  const VerifyLayout L = verify_layout(MODE, BV, F32IN ? 4 : 2, a.tm);
  const int grp = a.Hv / a.Hk;
  const long nshare = (long)a.batch * a.Hk;
  const long blocks = 8 * ((nshare + 7) / 8) * grp * NSL;
  if (blocks == 0) return TL_OK;
  if (blocks > 0x7fffffffL) return TL_EINVAL;
  auto kern = verify_kernel<MODE, D, BV, F32IN>;
  if (L.total > 64 * 1024) {
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                            hipFuncAttributeMaxDynamicSharedMemorySize, L.total) != hipSuccess)
      return TL_EHIP;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kThreads), L.total, stream, a);
  return hipGetLastError() == hipSuccess ? TL_OK : TL_EHIP;
}

template <int MODE, bool F32IN>
static tl_status dispatch_d(int d, const VerifyArgs& a, hipStream_t stream) {
  switch (d) {
    case 16: return launch_one<MODE, 16, 16, F32IN>(a, stream);
    case 32: return launch_one<MODE, 32, 32, F32IN>(a, stream);
    case 64: return launch_one<MODE, 64, 64, F32IN>(a, stream);
    case 128: return launch_one<MODE, 128, (MODE == TL_MODE_GDN ? 64 : 128), F32IN>(a, stream);
    default: return TL_EUNSUPPORTED;
  }
}

tl_status launch_verify(const tl_problem& p, const VerifyArgs& a, hipStream_t stream) {
  if (p.mode == TL_MODE_GLA)
    return p.in_dtype == TL_F32 ? dispatch_d<TL_MODE_GLA, true>(p.d_k, a, stream)
                                : dispatch_d<TL_MODE_GLA, false>(p.d_k, a, stream);
  return p.in_dtype == TL_F32 ? dispatch_d<TL_MODE_GDN, true>(p.d_k, a, stream)
                              : dispatch_d<TL_MODE_GDN, false>(p.d_k, a, stream);
}

int verify_lds_bytes(const tl_problem& p, int tm) {
  const int bv = (p.mode == TL_MODE_GDN && p.d_v == 128) ? 64 : p.d_v;
  return verify_layout(p.mode, bv, p.in_dtype == TL_F32 ? 4 : 2, tm).total;
}

}  // namespace tl
