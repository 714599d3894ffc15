// Verify, gated linear attention on MFMA.
//
// One workgroup handles one (request b, v-head h, value slice).  Q, K and the
// state slice arrive by direct global -> LDS copies and loads into MFMA operand
// registers, V^T is staged through registers, and after one barrier every wave
// works through the node tiles on its own value rows.
//
// For node tile I (16 nodes, columns i) a wave computes, for its value rows v,
//   O^T = P .* (S Q_I^T)  +  V^T C_I^T,   C_ij = [j in Anc(i) u {i}] 2^(cl_i - cl_j) (k_j . q_i)
// with cl the cumulative log-decay along the root path in log2 units.  The
// tree term runs over 32-node chunks of j: the MFMA K_J Q_I^T returns row
// j = 4*(l/16)+r of column i = l%16 in lane l, which is exactly the element of
// C^T that lane l supplies as the B operand of V^T C^T in the kpos() layout.
// So C is masked, decayed, split into bf16 hi + lo and consumed by the next
// MFMA without leaving registers, and the waves never wait for each other
// inside the tile loop.  The state is split into bf16 hi + lo as well, so both
// products keep ~2^-17 relative accuracy with bf16 MFMA.
#pragma once

#include "verify_common.h"

namespace tl {

struct GlaLayout {
  int x, cl, mask, tmask, qst, kst, vt, total;
};

// V^T row stride (elements): the tree term reads whole 32-node chunks, so
// rows hold 32 * ceil(tm / 32) columns, plus 8: stride / 2 = 4 (mod 8) 32-bit
// words, so the 8-byte fragment reads of 16 rows by 4 lane groups hit 64
// different banks.
__host__ __device__ constexpr int gla_vt_stride(int tm) { return ((tm + 31) & ~31) + 8; }

// C operand fragments of a tree of nt node tiles (trees of <= 64 nodes): tile
// I uses I / 2 + 1 chunks of 32 ancestor columns.
__host__ __device__ constexpr int gla_small_slots(int nt) { return (nt * nt + 2 * nt + (nt & 1)) / 4; }

// LDS layout of the MFMA paths (bytes).
__host__ __device__ inline GlaLayout gla_layout(int D, int BV, int tm, int W) {
  GlaLayout L;
  int o = 0;
  L.x = o;     o += align16(tm * 4);                     // log-decay inputs x = g
  L.cl = o;    o += align16((tm + 32) * 4);              // cumulative log2-decay (+1 chunk pad)
  L.mask = o;  o += tm * W * 8;                          // M+ rows
  L.tmask = o; o += align16((tm / kTile) * W * 8);       // OR of M+ rows per node tile
  L.qst = o;   o += (W == 1) ? tm * D * 2 : 0;           // Q rows (trees of <= 64 nodes)
  L.kst = o;   o += tm * D * 2;                          // K rows, swizzled bf16
  L.vt = o;                                              // V^T [BV][stride] bf16
  const int vt = BV * gla_vt_stride(tm) * 2;
  const int topo = kThreads * (4 + 4 + 4) + kThreads * W * 8;   // aliases V^T (prologue only)
  o += align16(vt > topo ? vt : topo);
  L.total = o;
  return L;
}

template <int D, int BV, int W>
__device__ inline void verify_gla_mfma(const VerifyArgs& a, const Unit u) {
  constexpr int KS = D / 32;
  constexpr int MTILES = BV / kTile;
  constexpr int MT = (MTILES + kWaves - 1) / kWaves;
  constexpr int CPRK = D / 8;
  constexpr bool QST = (W == 1);
  constexpr int VCH = BV / 8;                                            // 16-byte chunks per value row
  constexpr int VTN = ((64 * W / 2) * VCH + kThreads - 1) / kThreads;    // V^T tasks per thread
  constexpr float kLog2e = 1.4426950408889634f;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, lr = lane & 15, lg = lane >> 4;
  const int T = u.T, off = u.off, hq = u.hq, tm = u.tm, slice = u.slice;
  const int TS = gla_vt_stride(tm);
  const GlaLayout L = gla_layout(D, BV, tm, W);
  float* s_x = reinterpret_cast<float*>(tl_lds + L.x);
  float* s_cl = reinterpret_cast<float*>(tl_lds + L.cl);
  uint64_t* s_mask = reinterpret_cast<uint64_t*>(tl_lds + L.mask);
  uint64_t* s_tmask = reinterpret_cast<uint64_t*>(tl_lds + L.tmask);
  __bf16* s_q = reinterpret_cast<__bf16*>(tl_lds + L.qst);
  __bf16* s_k = reinterpret_cast<__bf16*>(tl_lds + L.kst);
  __bf16* s_vt = reinterpret_cast<__bf16*>(tl_lds + L.vt);
  int* s_flag = reinterpret_cast<int*>(s_x);

  const size_t qk_row = (size_t)a.Hk * D, v_row = (size_t)a.Hv * D;
  const __bf16* Qb = reinterpret_cast<const __bf16*>(a.q) + (size_t)off * qk_row + (size_t)hq * D;
  const __bf16* Kb = reinterpret_cast<const __bf16*>(a.k) + (size_t)off * qk_row + (size_t)hq * D;
  const int h0 = u.h;
  const float* Sbase = a.state + (size_t)u.sidx * a.Hv * D * D + (size_t)slice * BV * D;

  // V rows of head h -> registers: task x = (node pair p, 8-column chunk cc)
  const int npair = (T + 1) >> 1;
  const int ntask = npair * VCH;
  auto load_v = [&](int h, bf16x8 (&v0)[VTN], bf16x8 (&v1)[VTN]) {
    const __bf16* Vb = reinterpret_cast<const __bf16*>(a.v) + (size_t)off * v_row + (size_t)h * D + slice * BV;
#pragma unroll
    for (int k = 0; k < VTN; ++k) {
      const int x = tid + k * kThreads;
      v0[k] = bf16x8{};
      v1[k] = bf16x8{};
      if (x < ntask) {
        const int p = x % npair, cc = x / npair;
        v0[k] = *reinterpret_cast<const bf16x8*>(Vb + (size_t)(2 * p) * v_row + cc * 8);
        if (2 * p + 1 < T) v1[k] = *reinterpret_cast<const bf16x8*>(Vb + (size_t)(2 * p + 1) * v_row + cc * 8);
      }
    }
  };
  // ... and from registers into V^T (two nodes per 32-bit word)
  auto store_vt = [&](const bf16x8 (&v0)[VTN], const bf16x8 (&v1)[VTN]) {
#pragma unroll
    for (int k = 0; k < VTN; ++k) {
      const int x = tid + k * kThreads;
      if (x < ntask) {
        const int p = x % npair, cc = x / npair;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const __bf16 pr[2] = {v0[k][e], v1[k][e]};
          *reinterpret_cast<uint32_t*>(s_vt + (size_t)(cc * 8 + e) * TS + 2 * p) =
              *reinterpret_cast<const uint32_t*>(pr);
        }
      }
    }
  };
  // state rows of head h -> registers, in MFMA A-operand layout (rows = value channels)
  auto load_s = [&](int h, f32x4 (&sr)[MT][KS][2]) {
    const float* Sp = Sbase + (size_t)h * D * D;
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const int mt = wave + kWaves * m;
      if (mt < MTILES) {
        const float* row = Sp + (size_t)(kTile * mt + lr) * D;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          sr[m][ks][0] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(row + ks * 32 + 4 * lg));
          sr[m][ks][1] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(row + ks * 32 + 16 + 4 * lg));
        }
      }
    }
  };

  // ---- 1. loads: parents and gates, the first head's state, Q / K into LDS, V rows
  TL_TRACE_POINT(a, 1);
  const int par = (tid < T) ? a.parent[off + tid] : -1;
  float gx = (tid < T) ? a.g[(size_t)(off + tid) * a.Hv + h0] : 0.f;
  f32x4 sraw[MT][KS][2];
  load_s(h0, sraw);
  stage_rows_bf16<CPRK>(Kb, qk_row, T, s_k);
  if constexpr (QST) stage_rows_bf16<CPRK>(Qb, qk_row, T, s_q);
  bf16x8 vr0[VTN], vr1[VTN];
  load_v(h0, vr0, vr1);

  // ---- 2. topology: M+ rows and their per-tile OR
  TL_TRACE_POINT(a, 2);
  {
    int dep = 0;
    float cl = 0.f;
    uint64_t msk[W];
#pragma unroll
    for (int w = 0; w < W; ++w) msk[w] = 0ull;
    bool ok;
    if (T <= 64) {
      if (wave == 0) {   // one wavefront, lane = node: ballot + shuffle pointer jumping
        uint64_t m1;
        ok = wave_topology(par, T, 0.f, dep, cl, m1);
        if (lane == 0) s_flag[0] = ok ? 0 : 1;
        msk[0] = m1;
      }
      __syncthreads();
      ok = s_flag[0] == 0;
    } else {
      int* s_jmp = reinterpret_cast<int*>(tl_lds + L.vt);
      float* s_acc = reinterpret_cast<float*>(s_jmp + kThreads);
      int* s_cnt = reinterpret_cast<int*>(s_acc + kThreads);
      uint64_t* s_msk = reinterpret_cast<uint64_t*>(s_cnt + kThreads);
      ok = build_topology<W, true>(par, T, 0.f, s_jmp, s_acc, s_cnt, s_msk, dep, cl, msk);
    }
    if (!ok) {
      if (tid == 0) report(a.dev_err, TL_EBADTREE);
      wait_vmem();   // let the in-flight LDS copies land before the block retires
      return;
    }
    __syncthreads();   // flag and topology scratch are dead from here
    for (int x = tid; x < (tm / kTile) * W; x += kThreads) s_tmask[x] = 0;
    __syncthreads();
    const bool mine = (T <= 64) ? (wave == 0 && lane < T) : (tid < T);
    if (mine) {
#pragma unroll
      for (int w = 0; w < W; ++w) {
        s_mask[tid * W + w] = msk[w];
        if (msk[w]) atomicOr(reinterpret_cast<unsigned long long*>(&s_tmask[(tid / kTile) * W + w]),
                             (unsigned long long)msk[w]);
      }
    }
    // zero V^T columns T .. 32*ceil(T/32)-1 (the last chunk reads them; they
    // stay zero for every head since later heads write columns < 2*npair only)
    const int c0 = 2 * npair, c1 = (T + 31) & ~31;
    const int nw = (c1 - c0) >> 1;
    for (int x = tid; x < nw * BV; x += kThreads) {
      const int v = x / nw, w2 = x % nw;
      *reinterpret_cast<uint32_t*>(s_vt + (size_t)v * TS + c0 + 2 * w2) = 0u;
    }
  }

  // operand fragment of row R + lr (R a multiple of 16) for K chunk ks: the
  // row's swizzle key is lr & (CPRK-1), so both 8-byte pieces have fixed
  // per-lane offsets inside a 16-row block
  const int key = lr & (CPRK - 1);
  const int fo_row = lr * D * 2 + (lg & 1) * 8;
  const unsigned char* qbase = reinterpret_cast<const unsigned char*>(s_q);
  const unsigned char* kbase = reinterpret_cast<const unsigned char*>(s_k);
  auto frag_at = [&](const unsigned char* base, int R, int ks) {
    const unsigned char* p = base + R * D * 2 + fo_row;
    const bf16x4 x0 = *reinterpret_cast<const bf16x4*>(p + (((4 * ks + (lg >> 1)) ^ key) * 16));
    const bf16x4 x1 = *reinterpret_cast<const bf16x4*>(p + (((4 * ks + 2 + (lg >> 1)) ^ key) * 16));
    return bf16x8{x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
  };
  // V^T fragment of value tile mt for ancestor chunk c: row 16 mt + lr, columns 32c + 4lg (+16)
  int vo[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) vo[m] = ((kTile * (wave + kWaves * m) + lr) * TS + 4 * lg) * 2;
  const unsigned char* vtbase = reinterpret_cast<const unsigned char*>(s_vt);

  // ---- 3. cumulative log-decay, V^T, state split; then the node tiles
  {
    const int h = h0;
    // cumulative log-decay of head h: sum of x over the root path, root first
    if (tid < T) s_x[tid] = gx;
    __syncthreads();
    if (tid < T) {
      float cl = 0.f;
#pragma unroll
      for (int w = 0; w < W; ++w) {
        uint64_t bits = s_mask[tid * W + w];
        while (bits) {
          cl += s_x[64 * w + __builtin_ctzll(bits)];
          bits &= bits - 1;
        }
      }
      s_cl[tid] = cl * kLog2e;
    }
    store_vt(vr0, vr1);
    TL_TRACE_POINT(a, 3);
    wait_vmem();   // the direct-to-LDS copies of Q and K, the state and value rows
    __syncthreads();   // Q, K, V^T, masks and cl are in LDS; head h's state is in registers
    TL_TRACE_POINT(a, 4);

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

    bf16x8 qn[KS];
    if constexpr (!QST) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qn[ks] = frag_bf16(Qb + (size_t)lr * qk_row, ks, lg, lr < T);
    }
    TL_TRACE_POINT(a, 5);

    float* obase = a.out + (size_t)off * v_row + (size_t)h * D + slice * BV;
    for (int n0 = 0; n0 < T; n0 += kTile) {
      const int I = n0 / kTile;
      const int i = n0 + lr;
      const bool iv = i < T;
      bf16x8 qf[KS];
      if constexpr (QST) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) qf[ks] = frag_at(qbase, n0, ks);   // rows >= T only reach columns >= T
      } else {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) qf[ks] = qn[ks];
        if (n0 + kTile < T) {
          const int inext = i + kTile;
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) qn[ks] = frag_bf16(Qb + (size_t)inext * qk_row, ks, lg, inext < T);
        }
      }
      // a. B0^T = S Q_I^T, scaled per column by P_i
      f32x4 acc[MT];
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (wave + kWaves * m < MTILES) {
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            acc[m] = mfma16(shi[m][ks], qf[ks], acc[m]);
            acc[m] = mfma16(slo[m][ks], qf[ks], acc[m]);
          }
        }
      }
      uint64_t mi[W];
#pragma unroll
      for (int w = 0; w < W; ++w) mi[w] = iv ? s_mask[i * W + w] : 0ull;
      const float cli = iv ? s_cl[i] : 0.f;
      const float Pi = iv ? __builtin_amdgcn_exp2f(cli) : 0.f;
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[m] *= Pi;

      // b. tree term over 32-node chunks of ancestors: acc += V^T C^T
      uint64_t tmk[W];
#pragma unroll
      for (int w = 0; w < W; ++w) tmk[w] = s_tmask[I * W + w];
      for (int c = 0; 2 * c <= I; ++c) {
        uint64_t tw = tmk[0], mw = mi[0];                // 64-bit words holding chunk c
#pragma unroll
        for (int w = 1; w < W; ++w)
          if ((c >> 1) == w) { tw = tmk[w]; mw = mi[w]; }
        const unsigned bits = (unsigned)(tw >> ((c & 1) * 32));
        const bool need0 = (bits & 0xFFFFu) != 0;
        const bool need1 = (2 * c + 1 <= I) && ((bits >> 16) != 0);
        if (!need0 && !need1) continue;                     // uniform across the block
        f32x4 qk0 = f32x4{0.f, 0.f, 0.f, 0.f}, qk1 = qk0;
        if (need0) {                                        // rows j >= T are masked below
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) qk0 = mfma16(frag_at(kbase, 32 * c, ks), qf[ks], qk0);
        }
        if (need1) {
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) qk1 = mfma16(frag_at(kbase, 32 * c + 16, ks), qf[ks], qk1);
        }
        const f32x4 cl0 = *reinterpret_cast<const f32x4*>(s_cl + 32 * c + 4 * lg);
        const f32x4 cl1 = *reinterpret_cast<const f32x4*>(s_cl + 32 * c + 16 + 4 * lg);
        const unsigned mb = (unsigned)(mw >> ((c & 1) * 32)) >> (4 * lg);   // bit r: j = 32c+4lg+r
        bf16x8 chi, clo;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const bool b0 = (mb >> r) & 1u;
          const bool b1 = (mb >> (16 + r)) & 1u;
          const float c0 = b0 ? __builtin_amdgcn_exp2f(cli - cl0[r]) * qk0[r] : 0.f;
          const float c1 = b1 ? __builtin_amdgcn_exp2f(cli - cl1[r]) * qk1[r] : 0.f;
          __bf16 h0b, l0b, h1b, l1b;
          split_bf16(c0, h0b, l0b);
          split_bf16(c1, h1b, l1b);
          chi[r] = h0b;
          clo[r] = l0b;
          chi[4 + r] = h1b;
          clo[4 + r] = l1b;
        }
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          if (wave + kWaves * m < MTILES) {
            const unsigned char* vrow = vtbase + vo[m] + 64 * c;
            const bf16x4 x0 = *reinterpret_cast<const bf16x4*>(vrow);
            const bf16x4 x1 = *reinterpret_cast<const bf16x4*>(vrow + 32);
            const bf16x8 vf = bf16x8{x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
            acc[m] = mfma16(vf, chi, acc[m]);
            acc[m] = mfma16(vf, clo, acc[m]);
          }
        }
      }
      // c. store
      if (iv) {
        float* orow = obase + (size_t)i * v_row;
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          const int mt = wave + kWaves * m;
          if (mt < MTILES)
            __builtin_nontemporal_store(a.q_scale * acc[m], reinterpret_cast<f32x4*>(orow + kTile * mt + 4 * lg));
        }
      }
    }
  }
}

}  // namespace tl
