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
// steps with vector ALU products, in a separate function.
#include <hip/hip_runtime.h>

#include "tl_device.h"
#include "tl_kernels.h"

namespace tl {

extern __shared__ __align__(16) unsigned char tl_lds[];

// ---------------------------------------------------------------------------
// LDS layout (bytes); identical on host and device.
// ---------------------------------------------------------------------------
struct VerifyLayout {
  int par, depth, cl, beta, mask, tmask, kst, vst, ubuf, uni, total;
};

__host__ __device__ inline int align16(int x) { return (x + 15) & ~15; }

__host__ __device__ inline VerifyLayout verify_layout(int mode, int D, int BV, int vbytes, int tm,
                                                      int W, bool mfma) {
  const bool gdn = (mode == TL_MODE_GDN);
  VerifyLayout L;
  int o = 0;
  L.par = o;   o += align16(tm * 4);
  L.depth = o; o += align16(tm * 4);
  L.cl = o;    o += align16(tm * 4);
  L.beta = o;  o += gdn ? align16(tm * 4) : 0;
  L.mask = o;  o += tm * W * 8;
  L.tmask = o; o += align16((tm / kTile) * W * 8);
  L.kst = o;   o += mfma ? tm * D * 2 : 0;                 // K rows, swizzled bf16
  L.vst = o;   o += gdn ? 0 : tm * BV * vbytes;            // value slice (GLA)
  L.ubuf = o;  o += gdn ? tm * BV * 4 : 0;                 // U rows (delta rule)
  L.uni = o;
  // union: topology scratch | per-tile coefficients (c, and G for the delta rule)
  const int topo = kThreads * (4 + 4 + 4) + kThreads * W * 8;
  const int coef = kTile * tm * 4 * (gdn ? 2 : 1);
  o += align16(topo > coef ? topo : coef);
  L.total = o;
  return L;
}

struct Unit {
  int b, h, hq, slice, off, T, sidx, tm;
};

// ---------------------------------------------------------------------------
// Vector path: one request with vector ALU products (fp32 inputs, d = 16, or
// fewer than 16 nodes).  Its loops are kept rolled so that, inlined, it does
// not raise the register count of the MFMA path.
// ---------------------------------------------------------------------------
template <int MODE, int D, int BV, bool F32IN, int W>
__device__ inline void verify_vector(const VerifyArgs& a, const Unit u) {
  constexpr int MTILES = BV / kTile;
  constexpr int MT = (MTILES + kWaves - 1) / kWaves;
  constexpr bool GDN = (MODE == TL_MODE_GDN);
  using VT = typename std::conditional<F32IN, float, __bf16>::type;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, lr = lane & 15, lg = lane >> 4;
  const int T = u.T, off = u.off, h = u.h, hq = u.hq, tm = u.tm;
  const VerifyLayout L = verify_layout(MODE, D, BV, (int)sizeof(VT), tm, W, !F32IN && D >= 32);
  int* s_par = reinterpret_cast<int*>(tl_lds + L.par);
  int* s_depth = reinterpret_cast<int*>(tl_lds + L.depth);
  float* s_cl = reinterpret_cast<float*>(tl_lds + L.cl);
  float* s_beta = reinterpret_cast<float*>(tl_lds + L.beta);
  float* s_c = reinterpret_cast<float*>(tl_lds + L.uni);
  float* s_G = s_c + kTile * tm;
  VT* s_v = reinterpret_cast<VT*>(tl_lds + L.vst);
  float* s_u = reinterpret_cast<float*>(tl_lds + L.ubuf);
  const float* Sp = a.state + ((size_t)u.sidx * a.Hv + h) * D * D;
  const size_t qk_row = (size_t)a.Hk * D, v_row = (size_t)a.Hv * D;

  {
    const int par = (tid < T) ? a.parent[off + tid] : -1;
    const float gx = (tid < T) ? a.g[(size_t)(off + tid) * a.Hv + h] : 0.f;
    int dep;
    float cl;
    uint64_t msk[W];
    int* s_jmp = reinterpret_cast<int*>(tl_lds + L.uni);
    float* s_acc = reinterpret_cast<float*>(s_jmp + kThreads);
    int* s_cnt = reinterpret_cast<int*>(s_acc + kThreads);
    uint64_t* s_msk = reinterpret_cast<uint64_t*>(s_cnt + kThreads);
    if (!build_topology<W, false>(par, T, gx, s_jmp, s_acc, s_cnt, s_msk, dep, cl, msk)) {
      if (tid == 0) report(a.dev_err, TL_EBADTREE);
      return;
    }
    __syncthreads();   // scratch is dead from here
    if (tid < T) {
      s_par[tid] = par;
      s_depth[tid] = dep;
      s_cl[tid] = cl;
      if constexpr (GDN) s_beta[tid] = a.beta[(size_t)(off + tid) * a.Hv + h];
    }
  }
  if constexpr (!GDN) {
    for (int x = tid; x < T * BV; x += kThreads) {
      const int r = x / BV, c = x % BV;
      s_v[r * BV + c] = reinterpret_cast<const VT*>(a.v)[(size_t)(off + r) * v_row + (size_t)h * D +
                                                          u.slice * BV + c];
    }
  }
  __syncthreads();

  for (int n0 = 0; n0 < T; n0 += kTile) {
    const int i = n0 + lr;
    const bool iv = i < T;
    const int il = lr;
    const float cli = iv ? s_cl[i] : 0.f;
    const int di = iv ? s_depth[i] : 0;
    const float bi = (GDN && iv) ? s_beta[i] : 0.f;
    f32x4 acc[MT], acck[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
      acck[m] = acc[m];
      const int mt = wave + kWaves * m;
      if (mt >= MTILES || !iv) continue;
      const size_t qbase = (size_t)(off + i) * qk_row + (size_t)hq * D;
#pragma unroll 1
      for (int r = 0; r < 4; ++r) {
        const float* srow = Sp + (size_t)(u.slice * BV + kTile * mt + 4 * lg + r) * D;
        float sq = 0.f, sk = 0.f;
#pragma unroll 2
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
    // ancestor coefficients by direct dot products: thread -> (node, depth class)
    {
      const int vi = n0 + (tid & 15);
      if (vi < T) {
        const int dvi = s_depth[vi];
        const float clv = s_cl[vi];
        const float bv = GDN ? s_beta[vi] : 0.f;
        const size_t ibase = (size_t)(off + vi) * qk_row + (size_t)hq * D;
        for (int t = tid >> 4; t <= dvi; t += kThreads / 16) {
          int j = vi;
          for (int s = dvi; s > t; --s) j = s_par[j];
          const size_t jbase = (size_t)(off + j) * qk_row + (size_t)hq * D;
          float qk = 0.f, kk = 0.f;
#pragma unroll 2
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
    __syncthreads();

    const float Pi = iv ? __expf(cli) : 0.f;
    float* orow = a.out + (size_t)(off + i) * v_row + (size_t)h * D + u.slice * BV;
    if constexpr (!GDN) {
      for (int m = 0; m < MT; ++m) {
        const int mt = wave + kWaves * m;
        if (mt >= MTILES || !iv) continue;
        const int vl = kTile * mt + 4 * lg;
        f32x4 o = Pi * acc[m];
        int j = i, t = di;
        while (j >= 0) {
          const VT* vp = s_v + j * BV + vl;
          o += s_c[il * tm + t] * f32x4{(float)vp[0], (float)vp[1], (float)vp[2], (float)vp[3]};
          j = s_par[j];
          --t;
        }
        *reinterpret_cast<f32x4*>(orow + vl) = a.q_scale * o;
      }
    } else {
      f32x4 rr[MT];
      int mylev = -1;
      for (int m = 0; m < MT; ++m) {
        const int mt = wave + kWaves * m;
        rr[m] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (mt >= MTILES || !iv) continue;
        const int vl = kTile * mt + 4 * lg;
        const f32x4 vv =
            load4<F32IN>(a.v, (size_t)(off + i) * v_row + (size_t)h * D + u.slice * BV + vl);
        rr[m] = bi * (vv - Pi * acck[m]);
        int j = s_par[i], t = di - 1;
        while (j >= n0) { j = s_par[j]; --t; }
        while (j >= 0) {
          rr[m] -= s_G[il * tm + t] * *reinterpret_cast<const f32x4*>(s_u + j * BV + vl);
          j = s_par[j];
          --t;
        }
      }
      if (iv) {
        mylev = 0;
        for (int j = s_par[i]; j >= n0; j = s_par[j]) ++mylev;
      }
      for (int lev = 0; __syncthreads_or(mylev >= lev); ++lev) {
        if (mylev == lev) {
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
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// MFMA path: one request, bf16 inputs, at least 16 nodes.
// ---------------------------------------------------------------------------
template <int MODE, int D, int BV, int W>
__device__ inline void verify_mfma(const VerifyArgs& a, const Unit u) {
  constexpr int KS = D / 32;               // 32-wide K chunks of the MFMA
  constexpr int MTILES = BV / kTile;       // 16-row value tiles in the slice
  constexpr int MT = (MTILES + kWaves - 1) / kWaves;  // tiles per wave
  constexpr int CPRK = D / 8;              // 16-byte chunks per K row
  constexpr int CPRV = BV / 8;             // 16-byte chunks per value-slice row
  constexpr bool GDN = (MODE == TL_MODE_GDN);
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, lr = lane & 15, lg = lane >> 4;
  const int T = u.T, off = u.off, h = u.h, hq = u.hq, tm = u.tm, slice = u.slice;
  const VerifyLayout L = verify_layout(MODE, D, BV, 2, tm, W, true);
  float* s_cl = reinterpret_cast<float*>(tl_lds + L.cl);
  float* s_beta = reinterpret_cast<float*>(tl_lds + L.beta);
  uint64_t* s_mask = reinterpret_cast<uint64_t*>(tl_lds + L.mask);
  uint64_t* s_tmask = reinterpret_cast<uint64_t*>(tl_lds + L.tmask);
  __bf16* s_k = reinterpret_cast<__bf16*>(tl_lds + L.kst);
  __bf16* s_v = reinterpret_cast<__bf16*>(tl_lds + L.vst);
  float* s_u = reinterpret_cast<float*>(tl_lds + L.ubuf);
  float* s_c = reinterpret_cast<float*>(tl_lds + L.uni);
  float* s_G = s_c + kTile * tm;

  const size_t qk_row = (size_t)a.Hk * D, v_row = (size_t)a.Hv * D;
  const __bf16* Qb = reinterpret_cast<const __bf16*>(a.q) + (size_t)off * qk_row + (size_t)hq * D;
  const __bf16* Kb = reinterpret_cast<const __bf16*>(a.k) + (size_t)off * qk_row + (size_t)hq * D;
  const __bf16* Vb = reinterpret_cast<const __bf16*>(a.v) + (size_t)off * v_row + (size_t)h * D +
                     slice * BV;

  // ---- 1. loads: topology inputs, then the state, then K / V into LDS
  const int par = (tid < T) ? a.parent[off + tid] : -1;
  const float gx = (tid < T) ? a.g[(size_t)(off + tid) * a.Hv + h] : 0.f;
  float bx = 0.f;
  if constexpr (GDN) bx = (tid < T) ? a.beta[(size_t)(off + tid) * a.Hv + h] : 0.f;

  f32x4 sraw[MT][KS][2];
  const float* Sp = a.state + ((size_t)u.sidx * a.Hv + h) * D * D;
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
  stage_rows_bf16<CPRK>(Kb, qk_row, T, s_k);
  if constexpr (!GDN) stage_rows_bf16<CPRV>(Vb, v_row, T, s_v);

  // ---- 2. topology and cumulative log-decay of v-head h
  for (int x = tid; x < (tm / kTile) * W; x += kThreads) s_tmask[x] = 0;
  {
    int dep;
    float cl;
    uint64_t msk[W];
    int* s_jmp = reinterpret_cast<int*>(tl_lds + L.uni);
    float* s_acc = reinterpret_cast<float*>(s_jmp + kThreads);
    int* s_cnt = reinterpret_cast<int*>(s_acc + kThreads);
    uint64_t* s_msk = reinterpret_cast<uint64_t*>(s_cnt + kThreads);
    if (!build_topology<W, true>(par, T, gx, s_jmp, s_acc, s_cnt, s_msk, dep, cl, msk)) {
      if (tid == 0) report(a.dev_err, TL_EBADTREE);
      wait_vmem();   // let the in-flight LDS copies land before the block retires
      return;
    }
    __syncthreads();   // topology scratch is dead from here
    if (tid < T) {
      s_cl[tid] = cl;
      if constexpr (GDN) s_beta[tid] = bx;
#pragma unroll
      for (int w = 0; w < W; ++w) {
        s_mask[tid * W + w] = msk[w];
        if (msk[w]) atomicOr(reinterpret_cast<unsigned long long*>(&s_tmask[(tid / kTile) * W + w]),
                             (unsigned long long)msk[w]);
      }
    }
  }
  wait_vmem();
  __syncthreads();   // K / V in LDS, topology in LDS, state in registers

  // ---- split the state into bf16 hi/lo operands
  bf16x8 shi[MT][KS], slo[MT][KS];
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

  // Q fragments of the first tile
  bf16x8 qn[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) qn[ks] = frag_bf16(Qb + (size_t)lr * qk_row, ks, lg, lr < T);

  // ---- 3. node tiles
  for (int n0 = 0; n0 < T; n0 += kTile) {
    const int I = n0 / kTile;
    const int i = n0 + lr;            // this lane's node: column of every tile
    const bool iv = i < T;
    const int il = lr;
    bf16x8 qf[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = qn[ks];
    if (n0 + kTile < T) {             // prefetch the next tile's Q fragments
      const int inext = i + kTile;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qn[ks] = frag_bf16(Qb + (size_t)inext * qk_row, ks, lg, inext < T);
    }
    uint64_t mi[W];
#pragma unroll
    for (int w = 0; w < W; ++w) mi[w] = iv ? s_mask[i * W + w] : 0ull;
    const float cli = iv ? s_cl[i] : 0.f;
    const float bi = (GDN && iv) ? s_beta[i] : 0.f;

    // a. B0^T = S Q^T (rows: value channels, columns: nodes), K S^T likewise
    bf16x8 kf[KS];
    if constexpr (GDN) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x4 x0 = lds_bf16x4<CPRK>(s_k, i, ks * 32 + 4 * lg);
        const bf16x4 x1 = lds_bf16x4<CPRK>(s_k, i, ks * 32 + 16 + 4 * lg);
        kf[ks] = iv ? bf16x8{x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]}
                    : bf16x8{};
      }
    }
    f32x4 acc[MT], acck[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
      acck[m] = acc[m];
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

    // b. ancestor coefficients from K Q^T (and K K^T) tiles
    {
      uint64_t tmk[W];
#pragma unroll
      for (int w = 0; w < W; ++w) tmk[w] = s_tmask[I * W + w];
      for (int J = wave; J <= I; J += kWaves) {
        const unsigned bits = (unsigned)((tmk[J >> 2] >> ((J & 3) * 16)) & 0xFFFFull);
        if (!bits) continue;                       // no ancestor of this tile in tile J
        const int jr = J * kTile + lr;
        f32x4 qk = f32x4{0.f, 0.f, 0.f, 0.f}, kk = qk;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x4 x0 = lds_bf16x4<CPRK>(s_k, jr, ks * 32 + 4 * lg);
          const bf16x4 x1 = lds_bf16x4<CPRK>(s_k, jr, ks * 32 + 16 + 4 * lg);
          const bf16x8 kj = (jr < T) ? bf16x8{x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]}
                                     : bf16x8{};
          qk = mfma16(kj, qf[ks], qk);             // rows j, column i: k_j . q_i
          if constexpr (GDN) kk = mfma16(kj, kf[ks], kk);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int j = J * kTile + 4 * lg + r;
          if (iv && ((mi[j >> 6] >> (j & 63)) & 1ull)) {
            const float dec = __expf(cli - s_cl[j]);
            const int t = popc_below<W>(mi, j);     // depth of ancestor j
            s_c[il * tm + t] = dec * qk[r];
            if constexpr (GDN) {
              if (j != i) s_G[il * tm + t] = bi * dec * kk[r];
            }
          }
        }
      }
    }
    __syncthreads();   // coefficients of this tile are in LDS

    const float Pi = iv ? __expf(cli) : 0.f;
    float* orow = a.out + (size_t)(off + i) * v_row + (size_t)h * D + slice * BV;

    if constexpr (!GDN) {
      // d. readout: O = P B0 + sum over the root path of c_ij v_j
      f32x4 o[MT];
#pragma unroll
      for (int m = 0; m < MT; ++m) o[m] = Pi * acc[m];
      if (iv) {
        int t = 0;
#pragma unroll
        for (int w = 0; w < W; ++w) {
          uint64_t bitsw = mi[w];
          while (bitsw) {
            const int j = 64 * w + __builtin_ctzll(bitsw);
            bitsw &= bitsw - 1;
            const float c = s_c[il * tm + t];
            ++t;
#pragma unroll
            for (int m = 0; m < MT; ++m) {
              const bf16x4 vv = lds_bf16x4<CPRV>(s_v, j, kTile * (wave + kWaves * m) + 4 * lg);
              o[m] += c * f32x4{(float)vv[0], (float)vv[1], (float)vv[2], (float)vv[3]};
            }
          }
        }
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          const int mt = wave + kWaves * m;
          if (mt < MTILES)
            *reinterpret_cast<f32x4*>(orow + kTile * mt + 4 * lg) = a.q_scale * o[m];
        }
      }
    } else {
      // c. R = beta (V - P (K S^T)), minus ancestors in earlier tiles (final)
      f32x4 rr[MT];
      const int t_n0 = popc_below<W>(mi, n0);     // ancestors before this tile
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        const int mt = wave + kWaves * m;
        rr[m] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (mt >= MTILES || !iv) continue;
        const int vl = kTile * mt + 4 * lg;
        const bf16x4 vv = *reinterpret_cast<const bf16x4*>(Vb + (size_t)i * v_row + vl);
        rr[m] = bi * (f32x4{(float)vv[0], (float)vv[1], (float)vv[2], (float)vv[3]} - Pi * acck[m]);
      }
      if (iv) {
        int t = 0;
#pragma unroll
        for (int w = 0; w < W; ++w) {
          uint64_t bitsw = mi[w];
          while (bitsw) {
            const int j = 64 * w + __builtin_ctzll(bitsw);
            if (j >= n0) break;
            bitsw &= bitsw - 1;
            const float gij = s_G[il * tm + t];
            ++t;
#pragma unroll
            for (int m = 0; m < MT; ++m)
              if (wave + kWaves * m < MTILES)
                rr[m] -= gij * *reinterpret_cast<const f32x4*>(s_u + j * BV + kTile * (wave + kWaves * m) + 4 * lg);
          }
        }
      }
      //    forward substitution inside the tile, one level at a time; the
      //    level of i is its number of strict ancestors inside the tile
      const int mylev = iv ? popc_below<W>(mi, i) - t_n0 : -1;
      for (int lev = 0; __syncthreads_or(mylev >= lev); ++lev) {
        if (mylev == lev) {
          int t = t_n0;
          for (int j = n0; j < i; ++j) {
            if (!((mi[j >> 6] >> (j & 63)) & 1ull)) continue;
            const float gij = s_G[il * tm + t];
            ++t;
#pragma unroll
            for (int m = 0; m < MT; ++m)
              if (wave + kWaves * m < MTILES)
                rr[m] -= gij * *reinterpret_cast<const f32x4*>(s_u + j * BV + kTile * (wave + kWaves * m) + 4 * lg);
          }
#pragma unroll
          for (int m = 0; m < MT; ++m)
            if (wave + kWaves * m < MTILES)
              *reinterpret_cast<f32x4*>(s_u + i * BV + kTile * (wave + kWaves * m) + 4 * lg) = rr[m];
        }
      }
      // d. readout: O = P B0 + sum over the root path of c_ij u_j
      if (iv) {
        f32x4 o[MT];
#pragma unroll
        for (int m = 0; m < MT; ++m) o[m] = Pi * acc[m];
        int t = 0;
#pragma unroll
        for (int w = 0; w < W; ++w) {
          uint64_t bitsw = mi[w];
          while (bitsw) {
            const int j = 64 * w + __builtin_ctzll(bitsw);
            bitsw &= bitsw - 1;
            const float c = s_c[il * tm + t];
            ++t;
#pragma unroll
            for (int m = 0; m < MT; ++m)
              if (wave + kWaves * m < MTILES)
                o[m] += c * *reinterpret_cast<const f32x4*>(s_u + j * BV + kTile * (wave + kWaves * m) + 4 * lg);
          }
        }
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          const int mt = wave + kWaves * m;
          if (mt < MTILES)
            *reinterpret_cast<f32x4*>(orow + kTile * mt + 4 * lg) = a.q_scale * o[m];
        }
      }
    }
    __syncthreads();   // the next tile rewrites the coefficients
  }
}

template <int MODE, int D, int BV, bool F32IN, int W>
__global__ __launch_bounds__(kThreads) void verify_kernel(VerifyArgs a) {
  constexpr int NSL = D / BV;              // value slices per head
  constexpr bool CAN_MFMA = !F32IN && D >= 32;
  const int tid = threadIdx.x;

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
  Unit u;
  u.b = sh / a.Hk;
  u.hq = sh % a.Hk;
  u.h = u.hq * grp + w_in / NSL;
  u.slice = w_in % NSL;
  u.tm = a.tm;

  Request rq;
  if (!load_request(a.node_offsets, u.b, a.max_nodes, a.dev_err, rq)) return;
  u.off = rq.off;
  u.T = rq.T;
  if (u.T == 0) return;
  u.sidx = a.slot ? a.slot[u.b] : u.b;
  if (u.sidx < 0 || u.sidx >= a.num_slots) {
    if (tid == 0) report(a.dev_err, TL_EINVAL);
    return;
  }
  if constexpr (CAN_MFMA) {
    if (u.T >= kTile) {
      verify_mfma<MODE, D, BV, W>(a, u);
      return;
    }
  }
  verify_vector<MODE, D, BV, F32IN, W>(a, u);
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
template <int MODE, int D, int BV, bool F32IN, int W>
static tl_status launch_one(const VerifyArgs& a, hipStream_t stream) {
  constexpr int NSL = D / BV;
  const VerifyLayout L = verify_layout(MODE, D, BV, F32IN ? 4 : 2, a.tm, W, !F32IN && D >= 32);
  const int grp = a.Hv / a.Hk;
  const long nshare = (long)a.batch * a.Hk;
  const long blocks = 8 * ((nshare + 7) / 8) * grp * NSL;
  if (blocks == 0) return TL_OK;
  if (blocks > 0x7fffffffL) return TL_EINVAL;
  auto kern = verify_kernel<MODE, D, BV, F32IN, W>;
  if (L.total > 64 * 1024) {
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                            hipFuncAttributeMaxDynamicSharedMemorySize, L.total) != hipSuccess)
      return TL_EHIP;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kThreads), L.total, stream, a);
  return hipGetLastError() == hipSuccess ? TL_OK : TL_EHIP;
}

template <int MODE, int D, int BV, bool F32IN>
static tl_status dispatch_w(const VerifyArgs& a, hipStream_t stream) {
  if (F32IN || a.tm > 128) return launch_one<MODE, D, BV, F32IN, 4>(a, stream);
  if (a.tm > 64) return launch_one<MODE, D, BV, F32IN, 2>(a, stream);
  return launch_one<MODE, D, BV, F32IN, 1>(a, stream);
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
  if (p.mode == TL_MODE_GLA)
    return p.in_dtype == TL_F32 ? dispatch_d<TL_MODE_GLA, true>(p.d_k, a, stream)
                                : dispatch_d<TL_MODE_GLA, false>(p.d_k, a, stream);
  return p.in_dtype == TL_F32 ? dispatch_d<TL_MODE_GDN, true>(p.d_k, a, stream)
                              : dispatch_d<TL_MODE_GDN, false>(p.d_k, a, stream);
}

}  // namespace tl
