// Verify, vector path: one (request, v-head, value slice) with vector ALU
// products.  Used for fp32 inputs, d = 16 and trees of fewer than 16 nodes.
#pragma once

#include "verify_common.h"

namespace tl {

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
  const VerifyLayout L = verify_layout(MODE, D, BV, (int)sizeof(VT), tm, W, false);
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

}  // namespace tl
