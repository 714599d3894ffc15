// Verify, gated linear attention on MFMA, trees of 16..64 nodes.
//
// Computes O^T = P .* (S Q^T) + V^T C^T per value tile (Theorem 1 with
// U = V), organised so that the coefficient matrix C is formed once per
// workgroup instead of once per wave, and so that a
// workgroup can serve NH = 1 or 2 v-heads that share a qk-head (grouped
// heads read the same q and k rows and the same tree, so K_J Q_I^T, the
// M+ rows and the q/k traffic are shared; only the gates, the values and the
// state differ):
//
//  prologue  wave 0 loads the parents and gates and runs the topology (M+
//            rows, cumulative log2-decay per head, per-tile OR of the M+ rows);
//            waves 1..3 copy the Q, K and V rows of every head straight into
//            swizzled row-major LDS (coalesced direct copies); V is read back
//            as the K-major MFMA operand by LDS transpose reads.
//            Every wave then requests head 0's state rows, which stream in
//            while the work that needs no state runs (the barriers
//            synchronise LDS only, so they do not wait for them).
//  (a)       the lower-triangular 16x16 blocks (I, J), J <= I, of
//            C_ij = [j in Anc(i) u {i}] 2^(cl_i - cl_j) (q_i . k_j) are spread
//            over the four waves; each block is one K_J Q_I^T MFMA chain whose
//            output lanes already hold the B-operand elements of V^T C^T, so
//            it is masked, decayed (per head) and split into bf16 hi + lo in
//            registers and written to LDS in operand order (over the dead K
//            rows).
//  per head  (c) the tree term V^T C^T from the stored operands, which needs
//            no state, then (b) S Q_I^T per node tile (state split into bf16
//            hi + lo) scaled by P_i and added, and the output.  Only the
//            state term waits for the head's state rows.
//
// A tree of <= 64 nodes has at most 4 node tiles, so C has at most 10
// blocks, kept as 6 operand fragments of 32 ancestor columns (hi and lo).
#pragma once

#include "verify_common.h"

namespace tl {

struct GlaSmallLayout {
  int cl, mask, tmask, flag, qst, kst, vst, total;
};

// LDS layout (bytes) of the <= 64-node path serving NH heads; identical on
// host and device.  C fragments of head h: slots [6h, 6h + 6) over the K rows.
__host__ __device__ inline GlaSmallLayout gla_small_layout(int D, int BV, int NH) {
  constexpr int tm = 64;
  GlaSmallLayout L;
  int o = 0;
  L.cl = o;    o += NH * (tm + 32) * 4;                 // cumulative log2-decay per head
  L.mask = o;  o += tm * 8;                             // M+ rows
  L.tmask = o; o += (tm / kTile) * 8;                   // OR of M+ rows per node tile
  L.flag = o;  o += 16;
  L.qst = o;   o += tm * D * 2;                         // Q rows, swizzled bf16
  L.kst = o;                                            // K rows | C fragments
  {
    const int kb = tm * D * 2;
    const int cb = NH * gla_small_slots(tm / kTile) * 2048;
    o += kb > cb ? kb : cb;
  }
  L.vst = o;   o += NH * tm * BV * 2;                   // V rows per head, swizzled bf16
  L.total = o;
  return L;
}

// Topology of a tree of T <= 64 nodes in one wavefront (lane = node): as
// wave_topology, accumulating NH per-node values along the root path (one
// cumulative log-decay per head).
template <int NH>
__device__ inline bool wave_topology_n(int par, int T, const float (&x)[NH], float (&cl)[NH],
                                       uint64_t& mask) {
  const int i = threadIdx.x & 63;
  const bool live = i < T;
  const bool bad = live && !(par == -1 || (par >= 0 && par < i));
  if (__ballot(bad)) return false;
  int jmp = live ? par : -1;
#pragma unroll
  for (int hh = 0; hh < NH; ++hh) cl[hh] = x[hh];
  mask = live ? (1ull << i) : 0ull;
  while (__ballot(jmp >= 0)) {
    const int src = jmp >= 0 ? jmp : i;
    const uint64_t m2 = shfl64(mask, src);
    const int j2 = __shfl(jmp, src, 64);
    float c2[NH];
#pragma unroll
    for (int hh = 0; hh < NH; ++hh) c2[hh] = __shfl(cl[hh], src, 64);
    if (jmp >= 0) {
      mask |= m2;
#pragma unroll
      for (int hh = 0; hh < NH; ++hh) cl[hh] += c2[hh];
      jmp = j2;
    }
  }
  return true;
}

template <int D, int BV, int NH>
__device__ inline void verify_gla_small(const VerifyArgs& a, const Unit u) {
  constexpr int KS = D / 32;
  constexpr int MTILES = BV / kTile;
  constexpr int MT = (MTILES + kWaves - 1) / kWaves;
  constexpr bool FULL = (MTILES % kWaves) == 0;   // every wave owns MT value tiles
  constexpr int CPRK = D / 8;
  constexpr int LT = kThreads - 64;               // loader threads (waves 1..3)
  static_assert(BV == D, "V rows are staged whole (one value slice per head)");
  constexpr int NTM = 4;                          // node tiles of a <= 64-node tree
  constexpr int NSLOT = gla_small_slots(NTM);     // C fragments per head
  constexpr int tm = 64;                          // the layout is always sized for 64 nodes
  constexpr float kLog2e = 1.4426950408889634f;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, lr = lane & 15, lg = lane >> 4;
  const int T = u.T, off = u.off, hq = u.hq, slice = u.slice, h0 = u.h;
  const GlaSmallLayout L = gla_small_layout(D, BV, NH);
  float* s_cl = reinterpret_cast<float*>(tl_lds + L.cl);   // [NH][tm + 32]
  uint64_t* s_mask = reinterpret_cast<uint64_t*>(tl_lds + L.mask);
  uint64_t* s_tmask = reinterpret_cast<uint64_t*>(tl_lds + L.tmask);
  int* s_flag = reinterpret_cast<int*>(tl_lds + L.flag);
  __bf16* s_q = reinterpret_cast<__bf16*>(tl_lds + L.qst);
  __bf16* s_k = reinterpret_cast<__bf16*>(tl_lds + L.kst);
  __bf16* s_v = reinterpret_cast<__bf16*>(tl_lds + L.vst);   // [NH][tm][BV]
  unsigned char* s_cf = tl_lds + L.kst;   // C operand fragments, over the K rows after (a)

  const size_t qk_row = (size_t)a.Hk * D, v_row = (size_t)a.Hv * D;
  const __bf16* Qb = reinterpret_cast<const __bf16*>(a.q) + (size_t)off * qk_row + (size_t)hq * D;
  const __bf16* Kb = reinterpret_cast<const __bf16*>(a.k) + (size_t)off * qk_row + (size_t)hq * D;

  // value tiles of this wave: MT adjacent tiles, so a wave writes whole
  // 128-byte output lines
  auto mtile = [&](int m) { return wave * MT + m; };
  auto has_tile = [&](int m) { return FULL || mtile(m) < MTILES; };

  // state rows of every head, in MFMA A-operand layout (rows = value channels).
  // Head 0's rows are requested right behind each wave's prologue loads and
  // copies, so that HBM streams the state while the tree is staged; the
  // prologue waits only for what was issued before them (vmcnt counts in
  // issue order).  Later heads' rows follow once the coefficients C are
  // formed, and each head's rows are waited for only by its state term.
  f32x4 sraw[NH][MT][KS][2];
  static_assert(FULL || MT == 1, "a wave owns all of its MT value tiles or none");
  auto load_state = [&](int hh) {
    issue_fence();
    __builtin_amdgcn_s_setprio(0);
    const float* Sp = a.state + ((size_t)u.sidx * a.Hv + h0 + hh) * D * D + (size_t)slice * BV * D;
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      if (!has_tile(m)) continue;
      const float* row = Sp + (size_t)(kTile * mtile(m) + lr) * D;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        sraw[hh][m][ks][0] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(row + ks * 32 + 8 * lg));
        sraw[hh][m][ks][1] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(row + ks * 32 + 8 * lg + 4));
      }
    }
    issue_fence();
  };
  // waits for every load and copy issued before load_state(0) (a wave that
  // owns no value tile issued no state loads)
  constexpr int NSL = (FULL ? MT : 1) * KS * 2;
  auto wait_before_state = [&]() {
    if (FULL || has_tile(0)) wait_vmem_below<NSL>();
    else wait_vmem();
  };
  // ---- prologue: loads, and the topology on wave 0.  Two workgroups share
  // a CU, and the older one's waves win the issue arbitration; the waves
  // issue their parents, gates and copies at raised priority and their state
  // rows at the normal one, so that both workgroups' copies enter the CU's
  // memory queue ahead of either's state rows and both can start on the
  // coefficients while the state streams in.
  __builtin_amdgcn_s_setprio(2);
  TL_TRACE_POINT(a, 1);
  int par = -1;
  float gx[NH];
#pragma unroll
  for (int hh = 0; hh < NH; ++hh) gx[hh] = 0.f;
  if (wave == 0) {   // lanes >= T read node 0 (in bounds; ignored by the topology)
    const int n = lane < T ? lane : 0;
    par = a.parent[off + n];
#pragma unroll
    for (int hh = 0; hh < NH; ++hh) gx[hh] = a.g[(size_t)(off + n) * a.Hv + h0 + hh];
    load_state(0);
    wait_before_state();
  }
  if (wave == 0) {
    float cl[NH];
    uint64_t m1 = 0ull;
    const bool ok = wave_topology_n<NH>(par, T, gx, cl, m1);
    uint64_t tor = m1;   // OR of the M+ rows of the lane's node tile
#pragma unroll
    for (int o = 1; o < kTile; o <<= 1) tor |= shfl64(tor, lane ^ o);
    if (lane == 0) s_flag[0] = ok ? 0 : 1;
    if (lane < T) {
      s_mask[lane] = m1;
#pragma unroll
      for (int hh = 0; hh < NH; ++hh) s_cl[hh * (tm + 32) + lane] = cl[hh] * kLog2e;
    }
    if (lr == 0) s_tmask[lane / kTile] = tor;
  } else {
    // Q and K rows straight into swizzled LDS: one wave instruction moves
    // 64 / CPRK whole rows; lane l always fills chunk position l % CPRK
    {
      constexpr int RPI = 64 / CPRK;        // rows per wave instruction
      constexpr int RSTEP = LT / CPRK;      // rows per step of the three waves
      const int cpos = lane % CPRK;
      const uint32_t rbytes = (uint32_t)(qk_row * 2);
      const char* kb = reinterpret_cast<const char*>(Kb);
      const char* qb = reinterpret_cast<const char*>(Qb);
      int r = (wave - 1) * RPI + lane / CPRK;
      for (int base = (wave - 1) * 64; base < T * CPRK; base += LT, r += RSTEP) {
        if (r < T) {
          const uint32_t so = (uint32_t)r * rbytes + (uint32_t)(swz<CPRK>(r, cpos) * 16);
          copy16_to_lds_async(kb + so, s_k + base * 8);
          copy16_to_lds_async(qb + so, s_q + base * 8);
        }
      }
    }
    // V rows of every head the same way, for the rows of every 32-node
    // chunk the tree term reads; rows past T repeat row T - 1 (finite values
    // that meet zero coefficients)
    {
      constexpr int RPI = 64 / CPRK;
      constexpr int RSTEP = LT / CPRK;
      const int cpos = lane % CPRK;
      const int TP = (T + 31) & ~31;
      const uint32_t rbytes = (uint32_t)(v_row * 2);
#pragma unroll
      for (int hh = 0; hh < NH; ++hh) {
        const char* vb = reinterpret_cast<const char*>(reinterpret_cast<const __bf16*>(a.v) + (size_t)off * v_row +
                                                       (size_t)(h0 + hh) * D);
        int r = (wave - 1) * RPI + lane / CPRK;
        for (int base = (wave - 1) * 64; base < TP * CPRK; base += LT, r += RSTEP) {
          const int rs = min(r, T - 1);
          const uint32_t so = (uint32_t)rs * rbytes + (uint32_t)(swz<CPRK>(r, cpos) * 16);
          copy16_to_lds_async(vb + so, s_v + (hh * tm * D) + base * 8);
        }
      }
    }
    load_state(0);
    wait_before_state();   // the direct-to-LDS copies, not the state
  }
  TL_TRACE_POINT(a, 3);
  lds_barrier();   // Q, K, V^T, M+ rows, tile masks and cl are in LDS
  if (s_flag[0] != 0) {
    if (tid == 0) report(a.dev_err, TL_EBADTREE);
    return;
  }
  TL_TRACE_POINT(a, 4);

  // operand fragment of row R + lr (R a multiple of 16), K chunk ks, from a
  // swizzled LDS matrix (fixed per-lane offsets inside a 16-row block)
  const int key = lr & (CPRK - 1);
  const int fo_row = lr * D * 2;
  auto frag_at = [&](const __bf16* base, int R, int ks) {
    const unsigned char* p = reinterpret_cast<const unsigned char*>(base) + R * D * 2 + fo_row;
    return *reinterpret_cast<const bf16x8*>(p + (((4 * ks + lg) ^ key) * 16));
  };

  // per-node values of the four node tiles, read once: M+ rows (zero for
  // nodes >= T) and cl of every head
  uint64_t mi[NTM];
  float cli[NH][NTM];
#pragma unroll
  for (int I = 0; I < NTM; ++I) {
    const int i = kTile * I + lr;
    const uint64_t mv = s_mask[i];
    mi[I] = i < T ? mv : 0ull;
#pragma unroll
    for (int hh = 0; hh < NH; ++hh) {
      const float cv = s_cl[hh * (tm + 32) + i];
      cli[hh][I] = i < T ? cv : 0.f;
    }
  }

  // ---- (a) C blocks (I, J), J <= I: block k = I (I + 1) / 2 + J goes to wave
  // k % 4.  Blocks are formed whether or not they hold an ancestor (the mask
  // zeroes them); rows and columns >= T are garbage in LDS and only ever
  // reach masked entries.
  constexpr int NB = 3;   // blocks per wave (10 blocks over 4 waves)
  uint32_t cw[NB][NH][4];   // coefficients (times q_scale) as bf16 pairs: hi01 hi23 lo01 lo23
#pragma unroll
  for (int kb = 0; kb < NB; ++kb) {
    const int k = min(wave + kWaves * kb, 9);
    const int I = (k >= 1) + (k >= 3) + (k >= 6);
    const int J = k - I * (I + 1) / 2;
    f32x4 qk = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qk = mfma16(frag_at(s_k, kTile * J, ks), frag_at(s_q, kTile * I, ks), qk);
    // this lane's M+ row for tile I, without dynamic register indexing
    uint64_t mrow = mi[0];
#pragma unroll
    for (int t = 1; t < NTM; ++t)
      if (I == t) mrow = mi[t];
    const unsigned mb = (unsigned)(mrow >> (kTile * J + 4 * lg)) & 0xFu;
#pragma unroll
    for (int hh = 0; hh < NH; ++hh) {
      float cl_i = cli[hh][0];
#pragma unroll
      for (int t = 1; t < NTM; ++t)
        if (I == t) cl_i = cli[hh][t];
      const f32x4 clj = *reinterpret_cast<const f32x4*>(s_cl + hh * (tm + 32) + kTile * J + 4 * lg);
      float c[4];
#pragma unroll
      for (int r = 0; r < 4; ++r)
        c[r] = ((mb >> r) & 1u) ? (__builtin_amdgcn_exp2f(cl_i - clj[r]) * a.q_scale) * qk[r] : 0.f;
      split2_bf16(c[0], c[1], cw[kb][hh][0], cw[kb][hh][2]);
      split2_bf16(c[2], c[3], cw[kb][hh][1], cw[kb][hh][3]);
    }
  }
  TL_TRACE_POINT(a, 5);
  lds_barrier();   // every wave is done with the K rows
  // fragments: [head][slot][hi | lo][lane] 16 bytes; block (I, J) fills half
  // J & 1 of slot (I, J / 2); the diagonal block of an even tile also zeroes
  // the other half (columns of tile I + 1, none of which is an ancestor)
#pragma unroll
  for (int kb = 0; kb < NB; ++kb) {
    const int k = wave + kWaves * kb;
    const int I = (k >= 1) + (k >= 3) + (k >= 6);
    const int J = k - I * (I + 1) / 2;
    if (k < 10) {
#pragma unroll
      for (int hh = 0; hh < NH; ++hh) {
        const int slot = hh * NSLOT + gla_small_slots(I) + (J >> 1);
        unsigned char* fh = s_cf + ((slot * 2) * 64 + lane) * 16;
        unsigned char* fl = fh + 64 * 16;
        *reinterpret_cast<uint2*>(fh + (J & 1) * 8) = uint2{cw[kb][hh][0], cw[kb][hh][1]};
        *reinterpret_cast<uint2*>(fl + (J & 1) * 8) = uint2{cw[kb][hh][2], cw[kb][hh][3]};
        if (J == I && (I & 1) == 0) {
          *reinterpret_cast<uint2*>(fh + 8) = uint2{0u, 0u};
          *reinterpret_cast<uint2*>(fl + 8) = uint2{0u, 0u};
        }
      }
    }
  }

  // transpose-read offsets: lane (lg, lr) names row 4 lg + lr / 4 of a
  // 16-node half chunk and columns 16 mt + 4 (lr % 4) .. + 3, so it receives
  // value channel 16 mt + lr of nodes 4 lg .. 4 lg + 3 (K positions kpos(lg, 0..3))
  const int vrow_l = 4 * lg + (lr >> 2);
  int vo[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    const int col = kTile * mtile(m) + 4 * (lr & 3);
    vo[m] = vrow_l * D * 2 + swz<CPRK>(vrow_l, col >> 3) * 16 + (col & 7) * 2;
  }
  f32x4 acc[NTM][MT];

  // tree term of head hh: acc = V^T (q_scale C)^T (needs no state)
  auto tree_term = [&](int hh) {
    const unsigned char* vbase = reinterpret_cast<const unsigned char*>(s_v + hh * tm * D);
#pragma unroll
    for (int I = 0; I < NTM; ++I) {
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[I][m] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c <= I / 2; ++c) {
        const int slot = hh * NSLOT + gla_small_slots(I) + c;
        const unsigned char* fh = s_cf + ((slot * 2) * 64 + lane) * 16;
        const bf16x8 chi = *reinterpret_cast<const bf16x8*>(fh);
        const bf16x8 clo = *reinterpret_cast<const bf16x8*>(fh + 64 * 16);
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          if (has_tile(m)) {
            // rows 32 c + vrow_l and 32 c + 16 + vrow_l keep the swizzle
            // key of row vrow_l (32 c and 16 are multiples of CPRK)
            const bf16x4 x0 = lds_read_tr16(vbase, vo[m] + (32 * c) * D * 2);
            const bf16x4 x1 = lds_read_tr16(vbase, vo[m] + (32 * c + 16) * D * 2);
            const bf16x8 vf = bf16x8{x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
            acc[I][m] = mfma16(vf, chi, acc[I][m]);
            acc[I][m] = mfma16(vf, clo, acc[I][m]);
          }
        }
      }
    }
  };
  // state term of head hh, then the output: per node tile,
  // O^T = acc + (q_scale P_i) S Q_I^T, with the state split into bf16 hi + lo;
  // Q rows >= T only reach output columns that are never stored
  auto state_term_and_store = [&](int hh) {
    bf16x8 shi[MT][KS], slo[MT][KS];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) split8_bf16(sraw[hh][m][ks][0], sraw[hh][m][ks][1], shi[m][ks], slo[m][ks]);
    float* obase = a.out + (size_t)off * v_row + (size_t)(h0 + hh) * D + slice * BV;
#pragma unroll
    for (int I = 0; I < NTM; ++I) {
      bf16x8 qf[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qf[ks] = frag_at(s_q, kTile * I, ks);
      f32x4 b0[MT];
#pragma unroll
      for (int m = 0; m < MT; ++m) b0[m] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int m = 0; m < MT; ++m)
          if (has_tile(m)) {
            b0[m] = mfma16(shi[m][ks], qf[ks], b0[m]);
            b0[m] = mfma16(slo[m][ks], qf[ks], b0[m]);
          }
      const float Pi = __builtin_amdgcn_exp2f(cli[hh][I]) * a.q_scale;
      const int i = kTile * I + lr;
      if (i < T) {
        float* orow = obase + (size_t)i * v_row;
#pragma unroll
        for (int m = 0; m < MT; ++m)
          if (has_tile(m))
            __builtin_nontemporal_store(acc[I][m] + Pi * b0[m], reinterpret_cast<f32x4*>(orow + kTile * mtile(m) + 4 * lg));
      }
    }
  };

#pragma unroll
  for (int hh = 1; hh < NH; ++hh) load_state(hh);
  lds_barrier();   // C fragments are in LDS
  TL_TRACE_POINT(a, 6);
#pragma unroll
  for (int hh = 0; hh < NH; ++hh) {
    tree_term(hh);               // while this head's state rows may still be arriving
    state_term_and_store(hh);
  }
}

}  // namespace tl
