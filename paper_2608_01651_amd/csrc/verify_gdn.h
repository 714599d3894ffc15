// Verify, delta rule on MFMA: one (request, v-head, value slice), node tiles
// in groups, U solved level by level in LDS.
#pragma once

#include "verify_common.h"

namespace tl {

// ---------------------------------------------------------------------------
// MFMA path: one request, bf16 inputs, at least 16 nodes.
//
// Nodes are handled in groups of NG = 256 / tm tiles of 16 (the whole tree
// when tm <= 64).  Per group: B0 (and K S^T) for every tile on MFMA, the
// ancestor coefficients of every node of the group (from K Q^T / K K^T tile
// pairs spread over the waves), one barrier, then (delta rule) a level-by-
// level solve over the group's depth range, and the readout.  A node has at
// most tm ancestors, so the coefficients of a group take NG*16*tm floats =
// 16 KB (another 16 KB for G).
// ---------------------------------------------------------------------------
template <int MODE, int D, int BV, int W>
__device__ inline void verify_gdn_mfma(const VerifyArgs& a, const Unit u) {
  constexpr int KS = D / 32;               // 32-wide K chunks of the MFMA
  constexpr int MTILES = BV / kTile;       // 16-row value tiles in the slice
  constexpr int MT = (MTILES + kWaves - 1) / kWaves;  // tiles per wave
  constexpr int CPRK = D / 8;              // 16-byte chunks per K row
  constexpr int CPRV = BV / 8;             // 16-byte chunks per value-slice row
  constexpr int NG = 4 / W;                // tiles per group: whole tree when tm <= 64
  constexpr bool QST = (W == 1);           // Q staged in LDS (else fragments from L2)
  constexpr bool GDN = (MODE == TL_MODE_GDN);
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, lr = lane & 15, lg = lane >> 4;
  const int T = u.T, off = u.off, h = u.h, hq = u.hq, tm = u.tm, slice = u.slice;
  const VerifyLayout L = verify_layout(MODE, D, BV, 2, tm, W, true);
  int* s_depth = reinterpret_cast<int*>(tl_lds + L.depth);
  float* s_cl = reinterpret_cast<float*>(tl_lds + L.cl);
  float* s_beta = reinterpret_cast<float*>(tl_lds + L.beta);
  uint64_t* s_mask = reinterpret_cast<uint64_t*>(tl_lds + L.mask);
  uint64_t* s_tmask = reinterpret_cast<uint64_t*>(tl_lds + L.tmask);
  int* s_misc = reinterpret_cast<int*>(tl_lds + L.par);      // [0] error flag, [1..2] depth range
  __bf16* s_q = reinterpret_cast<__bf16*>(tl_lds + L.qst);
  __bf16* s_k = reinterpret_cast<__bf16*>(tl_lds + L.kst);
  __bf16* s_v = reinterpret_cast<__bf16*>(tl_lds + L.vst);
  float* s_u = reinterpret_cast<float*>(tl_lds + L.ubuf);
  float* s_c = reinterpret_cast<float*>(tl_lds + L.uni);
  float* s_G = s_c + kTile * NG * tm;

  const size_t qk_row = (size_t)a.Hk * D, v_row = (size_t)a.Hv * D;
  const __bf16* Qb = reinterpret_cast<const __bf16*>(a.q) + (size_t)off * qk_row + (size_t)hq * D;
  const __bf16* Kb = reinterpret_cast<const __bf16*>(a.k) + (size_t)off * qk_row + (size_t)hq * D;
  const __bf16* Vb = reinterpret_cast<const __bf16*>(a.v) + (size_t)off * v_row + (size_t)h * D +
                     slice * BV;

  // ---- 1. loads: topology inputs, then the state, then K / V into LDS
  TL_TRACE_POINT(a, 1);
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
  if constexpr (QST) stage_rows_bf16<CPRK>(Qb, qk_row, T, s_q);
  if constexpr (!GDN) stage_rows_bf16<CPRV>(Vb, v_row, T, s_v);

  // ---- 2. topology and cumulative log-decay of v-head h
  TL_TRACE_POINT(a, 2);
  for (int x = tid; x < (tm / kTile) * W; x += kThreads) s_tmask[x] = 0;
  {
    int dep = 0;
    float cl = 0.f;
    uint64_t msk[W];
    bool ok;
    if (T <= 64) {
      // one wavefront, lane = node: ballot + shuffle pointer jumping
      if (wave == 0) {
        uint64_t m1;
        ok = wave_topology(par, T, gx, dep, cl, m1);
        if (lane == 0) s_misc[0] = ok ? 0 : 1;
#pragma unroll
        for (int w = 0; w < W; ++w) msk[w] = (w == 0) ? m1 : 0ull;
      }
      __syncthreads();
      ok = s_misc[0] == 0;
    } else {
      int* s_jmp = reinterpret_cast<int*>(tl_lds + L.uni);
      float* s_acc = reinterpret_cast<float*>(s_jmp + kThreads);
      int* s_cnt = reinterpret_cast<int*>(s_acc + kThreads);
      uint64_t* s_msk = reinterpret_cast<uint64_t*>(s_cnt + kThreads);
      ok = build_topology<W, true>(par, T, gx, s_jmp, s_acc, s_cnt, s_msk, dep, cl, msk);
    }
    if (!ok) {
      if (tid == 0) report(a.dev_err, TL_EBADTREE);
      wait_vmem();   // let the in-flight LDS copies land before the block retires
      return;
    }
    __syncthreads();   // topology scratch is dead from here
    const bool mine = (T <= 64) ? (wave == 0 && lane < T) : (tid < T);
    if (mine) {
      s_depth[tid] = dep;
      s_cl[tid] = cl;
#pragma unroll
      for (int w = 0; w < W; ++w) {
        s_mask[tid * W + w] = msk[w];
        if (msk[w]) atomicOr(reinterpret_cast<unsigned long long*>(&s_tmask[(tid / kTile) * W + w]),
                             (unsigned long long)msk[w]);
      }
    }
    if constexpr (GDN) {
      if (tid < T) s_beta[tid] = bx;
    }
  }
  TL_TRACE_POINT(a, 3);
  wait_vmem();
  __syncthreads();   // K / V in LDS, topology in LDS, state in registers
  TL_TRACE_POINT(a, 4);

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

  // Q fragments of the first tile (when Q is not staged)
  bf16x8 qn[KS];
  if constexpr (!QST) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qn[ks] = frag_bf16(Qb + (size_t)lr * qk_row, ks, lg, lr < T);
  }
  TL_TRACE_POINT(a, 5);

  // ---- 3. groups of NG node tiles
  for (int g0 = 0; g0 < T; g0 += NG * kTile) {
    const int I0 = g0 / kTile;
    if constexpr (GDN) {
      if (tid == 0) { s_misc[1] = 1 << 30; s_misc[2] = -1; }
    }
    f32x4 acc[NG][MT];
    uint64_t mi[NG][W];
#pragma unroll
    for (int ig = 0; ig < NG; ++ig) {
      const int n0 = g0 + ig * kTile;
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[ig][m] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int w = 0; w < W; ++w) mi[ig][w] = 0ull;
      if (n0 >= T) continue;                    // uniform
      const int I = I0 + ig;
      const int i = n0 + lr;                    // this lane's node: column of every tile
      const bool iv = i < T;
      const int il = ig * kTile + lr;           // node index inside the group
      bf16x8 qf[KS];
      if constexpr (QST) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) qf[ks] = lds_frag<CPRK>(s_q, i, ks, lg, iv);
      } else {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) qf[ks] = qn[ks];
        if (n0 + kTile < T) {                   // prefetch the next tile's Q fragments
          const int inext = i + kTile;
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            qn[ks] = frag_bf16(Qb + (size_t)inext * qk_row, ks, lg, inext < T);
        }
      }
#pragma unroll
      for (int w = 0; w < W; ++w) mi[ig][w] = iv ? s_mask[i * W + w] : 0ull;
      const float cli = iv ? s_cl[i] : 0.f;
      const float bi = (GDN && iv) ? s_beta[i] : 0.f;

      // a. B0^T = S Q^T (rows: value channels, columns: nodes), K S^T likewise
      bf16x8 kf[KS];
      if constexpr (GDN) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) kf[ks] = lds_frag<CPRK>(s_k, i, ks, lg, iv);
      }
      f32x4 acck[MT];
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        acck[m] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (wave + kWaves * m < MTILES) {
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            acc[ig][m] = mfma16(shi[m][ks], qf[ks], acc[ig][m]);
            acc[ig][m] = mfma16(slo[m][ks], qf[ks], acc[ig][m]);
            if constexpr (GDN) {
              acck[m] = mfma16(shi[m][ks], kf[ks], acck[m]);
              acck[m] = mfma16(slo[m][ks], kf[ks], acck[m]);
            }
          }
        }
      }
      if constexpr (GDN) {
        // R = beta (V - P (K S^T)) -> U rows (solved in place below)
        const float Pi = iv ? __expf(cli) : 0.f;
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          const int mt = wave + kWaves * m;
          if (mt < MTILES && iv) {
            const int vl = kTile * mt + 4 * lg;
            const bf16x4 vv = *reinterpret_cast<const bf16x4*>(Vb + (size_t)i * v_row + vl);
            *reinterpret_cast<f32x4*>(s_u + i * BV + vl) =
                bi * (f32x4{(float)vv[0], (float)vv[1], (float)vv[2], (float)vv[3]} - Pi * acck[m]);
          }
        }
        if (iv && wave == 0 && lg == 0) {
          atomicMin(&s_misc[1], s_depth[i]);
          atomicMax(&s_misc[2], s_depth[i]);
        }
      }

      // b. ancestor coefficients from K Q^T (and K K^T) tiles; the I+1 tile
      //    pairs (I, J <= I) are dealt round robin over the waves
      uint64_t tmk[W];
#pragma unroll
      for (int w = 0; w < W; ++w) tmk[w] = s_tmask[I * W + w];
      const int first = (wave - (I * (I + 1) / 2) % kWaves + kWaves) % kWaves;
      for (int J = first; J <= I; J += kWaves) {
        const unsigned bits = (unsigned)((tmk[J >> 2] >> ((J & 3) * 16)) & 0xFFFFull);
        if (!bits) continue;                     // no ancestor of this tile in tile J
        const int jr = J * kTile + lr;
        f32x4 qk = f32x4{0.f, 0.f, 0.f, 0.f}, kk = qk;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8 kj = lds_frag<CPRK>(s_k, jr, ks, lg, jr < T);
          qk = mfma16(kj, qf[ks], qk);             // rows j, column i: k_j . q_i
          if constexpr (GDN) kk = mfma16(kj, kf[ks], kk);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int j = J * kTile + 4 * lg + r;
          if (iv && ((mi[ig][j >> 6] >> (j & 63)) & 1ull)) {
            const float dec = __expf(cli - s_cl[j]);
            const int t = popc_below<W>(mi[ig], j);     // depth of ancestor j
            s_c[il * tm + t] = dec * qk[r];
            if constexpr (GDN) {
              if (j != i) s_G[il * tm + t] = bi * dec * kk[r];
            }
          }
        }
      }
    }
    __syncthreads();   // coefficients (and R) of the group are in LDS
    if (g0 < 4 * NG * kTile) TL_TRACE_POINT(a, 6 + 2 * (g0 / (NG * kTile)));

    if constexpr (GDN) {
      // c. forward substitution of (I + G) U = R, one depth level at a time:
      //    a node at depth d subtracts G_ij u_j over its strict ancestors, all
      //    of which sit at smaller depths (earlier groups or earlier levels)
      const int dlo = s_misc[1], dhi = s_misc[2];
      for (int lev = dlo; lev <= dhi; ++lev) {
#pragma unroll
        for (int ig = 0; ig < NG; ++ig) {
          const int i = g0 + ig * kTile + lr;
          if (i >= T || s_depth[i] != lev) continue;
          const int il = ig * kTile + lr;
#pragma unroll
          for (int m = 0; m < MT; ++m) {
            const int mt = wave + kWaves * m;
            if (mt >= MTILES) continue;
            const int vl = kTile * mt + 4 * lg;
            f32x4 r = *reinterpret_cast<const f32x4*>(s_u + i * BV + vl);
            int tb = 0;   // strict ancestors in earlier mask words
#pragma unroll
            for (int w = 0; w < W; ++w) {
              uint64_t bitsw = mi[ig][w];
              if (64 * w <= i && i < 64 * w + 64) bitsw &= ~(1ull << (i & 63));   // strict ancestors
              int t = tb;
              tb += __popcll(bitsw);
              while (bitsw) {   // four ancestors per round trip
                int jj[4];
                float gg[4];
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                  const bool have = bitsw != 0;
                  jj[q4] = have ? 64 * w + __builtin_ffsll((long long)bitsw) - 1 : i;
                  gg[q4] = have ? s_G[il * tm + min(t + q4, tm - 1)] : 0.f;
                  bitsw &= bitsw - 1;
                }
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4)
                  r -= gg[q4] * *reinterpret_cast<const f32x4*>(s_u + jj[q4] * BV + vl);
                t += 4;
              }
            }
            *reinterpret_cast<f32x4*>(s_u + i * BV + vl) = r;
          }
        }
        __syncthreads();
      }
    }

    if (g0 < 4 * NG * kTile) TL_TRACE_POINT(a, 7 + 2 * (g0 / (NG * kTile)));
    // d. readout: O = P B0 + sum over the root path of c_ij u_j  (u = v for GLA)
#pragma unroll
    for (int ig = 0; ig < NG; ++ig) {
      const int i = g0 + ig * kTile + lr;
      if (g0 + ig * kTile >= T || i >= T) continue;
      const int il = ig * kTile + lr;
      const float Pi = __expf(s_cl[i]);
      f32x4 o[MT];
#pragma unroll
      for (int m = 0; m < MT; ++m) o[m] = Pi * acc[ig][m];
      int tb = 0;   // ancestors (and self) in earlier mask words
#pragma unroll
      for (int w = 0; w < W; ++w) {
        uint64_t bitsw = mi[ig][w];
        int t = tb;
        tb += __popcll(bitsw);
        while (bitsw) {   // four ancestors per round trip
          int jj[4];
          float cc[4];
#pragma unroll
          for (int q4 = 0; q4 < 4; ++q4) {
            const bool have = bitsw != 0;
            jj[q4] = have ? 64 * w + __builtin_ffsll((long long)bitsw) - 1 : i;
            cc[q4] = have ? s_c[il * tm + min(t + q4, tm - 1)] : 0.f;
            bitsw &= bitsw - 1;
          }
          t += 4;
#pragma unroll
          for (int q4 = 0; q4 < 4; ++q4) {
#pragma unroll
            for (int m = 0; m < MT; ++m) {
              const int vl = kTile * (wave + kWaves * m) + 4 * lg;
              if constexpr (GDN) {
                o[m] += cc[q4] * *reinterpret_cast<const f32x4*>(s_u + jj[q4] * BV + vl);
              } else {
                const bf16x4 vv = lds_bf16x4<CPRV>(s_v, jj[q4], vl);
                o[m] += cc[q4] * f32x4{(float)vv[0], (float)vv[1], (float)vv[2], (float)vv[3]};
              }
            }
          }
        }
      }
      float* orow = a.out + (size_t)(off + i) * v_row + (size_t)h * D + slice * BV;
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        const int mt = wave + kWaves * m;
        if (mt < MTILES) *reinterpret_cast<f32x4*>(orow + kTile * mt + 4 * lg) = a.q_scale * o[m];
      }
    }
    __syncthreads();   // the next group rewrites the coefficients
  }
}

}  // namespace tl
