// Verify on MFMA, node tile by node tile: the gated delta rule wherever its
// tile-sequential layout fits in LDS and the dense kernel does not serve it
// (node caps of 129..160 at d = 128, and d = 32, 64).
//
// One workgroup per (request, v-head) with one wave per 16-row value tile
// of the stored state (8 waves at d = 128).  Nodes are taken in tiles of 16
// in index order, which is topological, so every ancestor of tile I lies in
// tiles 0..I.  For tile I:
//
//  1. coefficients: the ancestor columns of tile I are cut into chunks of
//     32 nodes (tiles 2c, 2c + 1).  The waves share the chunks; a chunk is
//     one K_J Q_I^T (and K_J K_I^T) MFMA chain per half, whose output lanes
//     hold the B-operand elements of U^T C^T, so it is masked, decayed and
//     split into bf16 hi + lo in registers and stored in operand order:
//       C_ij = [j in Anc(i) u {i}] 2^(cl_i - cl_j) (q_i . k_j) q_scale
//       G_ij = [j in Anc(i)]       beta_i 2^(cl_i - cl_j) (k_i . k_j)
//     (Theorem 1, Lemma 2; cl = cumulative log2-decay).  The block of G
//     inside tile I goes to a small row-major array instead.
//  2. delta rule: per wave (its value rows v), in MFMA output layout,
//       X = beta (V - P (S K_I^T))               (R of Lemma 2)
//       X -= U^T G^T over the chunks of earlier tiles (MFMA, U in hi + lo)
//     then the in-tile part of (I + G) U = R by forward substitution over
//     the few in-tile ancestors (u_j broadcast along each 16-lane row by
//     DPP), and U_I^T goes to LDS as
//     bf16 hi + lo.  Only the wave's own rows of U^T are ever read back, so
//     the solve needs no barrier: (I + G) is unit lower triangular and the
//     tiles are solved in order (Lemma 3 bounds the depth, not needed here).
//  3. readout: O^T = q_scale P_i (S Q_I^T) + U^T C^T, stored as fp32.
//
// When LDS holds two chunk buffers, the coefficients of tile I + 1 are
// formed while tile I's value work runs, with one barrier per tile;
// otherwise the two phases alternate, with two.  The barriers order LDS
// only, so the Q and V rows, loaded two tiles ahead, and the output
// stores of the previous tile stay in flight across them.  The state is read
// once, split into bf16 hi + lo in registers.
#include <hip/hip_runtime.h>

#include "tl_device.h"
#include "tl_kernels.h"
#include "verify_common.h"

namespace tl {

__host__ __device__ constexpr int tiled_waves(int D) { return D / kTile > kWaves ? D / kTile : kWaves; }

struct TiledLayout {
  int cl, beta, mask, tmask, tin, gin, kst, frag, fragsz, frag2, ut, total;
};

// U^T row stride (elements): the value term reads whole 32-node chunks, so
// rows hold 32 * ceil(tm / 32) columns, plus 8: stride / 2 = 4 (mod 8)
// 32-bit words, so the 8-byte fragment reads of 16 rows by 4 lane groups hit
// 64 different banks.
__host__ __device__ constexpr int tiled_ut_stride(int tm) { return ((tm + 31) & ~31) + 8; }

// LDS layout (bytes); identical on host and device.  With db the chunk
// operands (and the in-tile block of G) are double-buffered.
__host__ __device__ inline TiledLayout tiled_layout(int D, int tm, int W, bool db) {
  const int nb = db ? 2 : 1;
  TiledLayout L;
  int o = 0;
  L.cl = o;    o += align16((tm + 32) * 4);                 // cumulative log2-decay (+1 chunk pad)
  L.beta = o;  o += align16(tm * 4);
  L.mask = o;  o += tm * W * 8;                             // M+ rows
  L.tmask = o; o += align16((tm / kTile) * W * 8);          // OR of M+ rows per node tile
  L.tin = o;   o += align16((tm / kTile) * 4);              // in-tile strict ancestors per tile
  L.gin = o;   o += nb * kTile * kTile * 4;                 // in-tile block of G, row-major
  L.kst = o;   o += tm * D * 2;                             // K rows, swizzled bf16
  L.frag = o;                                               // chunk operands | topology scratch
  L.fragsz = ((tm + 31) / 32) * 4 * 1024;                  // chunks of tiles 0..I, I < tm / 16
  {
    const int fr = nb * L.fragsz;
    const int topo = kThreads * (4 + 4 + 4) + kThreads * W * 8;
    o += align16(fr > topo ? fr : topo);
  }
  L.ut = o;    o += D * tiled_ut_stride(tm) * 2 * 2;        // U^T hi and lo
  L.frag2 = db ? L.frag + L.fragsz : L.frag;                // the second chunk buffer
  L.total = o;
  return L;
}

template <int D, int W, bool DB>
__global__ __launch_bounds__(64 * tiled_waves(D)) void verify_tiled_kernel(VerifyArgs a) {
  constexpr int NW = tiled_waves(D);
  constexpr int NT = 64 * NW;
  constexpr int VT = D / kTile;            // value tiles: wave w < VT owns rows 16w..16w+15
  constexpr int KS = D / 32;
  constexpr int CPRK = D / 8;
  constexpr int NF = 4;                    // 1 KB operand pieces per chunk: C hi, C lo, G hi, G lo
  constexpr float kLog2e = 1.4426950408889634f;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, lr = lane & 15, lg = lane >> 4;
  const bool vw = wave < VT;
  lds_poison(a.lds_bytes);
  TL_TRACE_POINT(a, 0);

  // ---- block -> (request, qk-head, v-head): the grouped v-heads of a qk-head
  // get ids 8 apart (same XCD, shared L2 for q/k)
  const int grp = a.Hv / a.Hk;
  const int nshare = a.batch * a.Hk;
  const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
  const int sh = (local / grp) * 8 + xcd;
  if (sh >= nshare) return;
  const int b = sh / a.Hk, hq = sh % a.Hk, h = hq * grp + local % grp;
  // the slot is read with the node range (independent loads, one round trip)
  const int sidx = a.slot ? a.slot[b] : b;
  Request rq;
  if (!load_request(a.node_offsets, b, a.max_nodes, a.dev_err, rq)) return;
  const int T = rq.T, off = rq.off;
  if (T == 0) return;
  if (sidx < 0 || sidx >= a.num_slots) {
    if (tid == 0) report(a.dev_err, TL_EINVAL);
    return;
  }
  const int tm = a.tm;
  const int TS = tiled_ut_stride(tm);
  const TiledLayout L = tiled_layout(D, tm, W, DB);
  float* s_cl = reinterpret_cast<float*>(tl_lds + L.cl);
  float* s_beta = reinterpret_cast<float*>(tl_lds + L.beta);
  uint64_t* s_mask = reinterpret_cast<uint64_t*>(tl_lds + L.mask);
  uint64_t* s_tmask = reinterpret_cast<uint64_t*>(tl_lds + L.tmask);
  uint32_t* s_tin = reinterpret_cast<uint32_t*>(tl_lds + L.tin);
  float* s_gin = reinterpret_cast<float*>(tl_lds + L.gin);
  __bf16* s_k = reinterpret_cast<__bf16*>(tl_lds + L.kst);
  unsigned char* s_frag = tl_lds + L.frag;
  __bf16* s_ut = reinterpret_cast<__bf16*>(tl_lds + L.ut);          // U^T hi
  __bf16* s_utl = s_ut + D * TS;                                      // U^T lo

  const size_t qk_row = (size_t)a.Hk * D, v_row = (size_t)a.Hv * D;
  const __bf16* Qb = reinterpret_cast<const __bf16*>(a.q) + (size_t)off * qk_row + (size_t)hq * D;
  const __bf16* Kb = reinterpret_cast<const __bf16*>(a.k) + (size_t)off * qk_row + (size_t)hq * D;
  const __bf16* Vb = reinterpret_cast<const __bf16*>(a.v) + (size_t)off * v_row + (size_t)h * D;

  // ---- prologue: parents and gates, the wave's state rows, K into LDS
  TL_TRACE_POINT(a, 1);
  int par = -1;
  float gx = 0.f, bx = 0.f;
  if (tid < T) {
    par = a.parent[off + tid];
    gx = a.g[(size_t)(off + tid) * a.Hv + h];
    bx = a.beta[(size_t)(off + tid) * a.Hv + h];
  }
  f32x4 sraw[KS][2];
  if (vw) {
    const float* row = a.state + ((size_t)sidx * a.Hv + h) * D * D + (size_t)(kTile * wave + lr) * D;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      sraw[ks][0] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(row + ks * 32 + 8 * lg));
      sraw[ks][1] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(row + ks * 32 + 8 * lg + 4));
    }
  }
  for (int base = wave * 64; base < T * CPRK; base += NT) {
    const int p = base + lane;
    if (p < T * CPRK) {
      const int r = p / CPRK, c = swz<CPRK>(r, p % CPRK);
      copy16_to_lds_async(Kb + (size_t)r * qk_row + c * 8, s_k + (size_t)base * 8);
    }
  }
  // U^T hi and lo start at zero: columns of later tiles are read (times zero
  // coefficients) before they are written
  {
    const int words = (D * TS * 2 * 2) / 16;
    for (int x = tid; x < words; x += NT) reinterpret_cast<uint4*>(s_ut)[x] = uint4{0u, 0u, 0u, 0u};
  }

  // ---- topology: M+ rows, cumulative log-decay, per-tile masks
  TL_TRACE_POINT(a, 2);
  for (int x = tid; x < (tm / kTile) * W; x += NT) s_tmask[x] = 0;
  for (int x = tid; x < tm / kTile; x += NT) s_tin[x] = 0u;
  {
    int* s_jmp = reinterpret_cast<int*>(s_frag);
    float* s_acc = reinterpret_cast<float*>(s_jmp + kThreads);
    int* s_cnt = reinterpret_cast<int*>(s_acc + kThreads);
    uint64_t* s_msk = reinterpret_cast<uint64_t*>(s_cnt + kThreads);
    int dep = 0;
    float cl = 0.f;
    uint64_t msk[W];
    const bool ok = build_topology<W, true>(par, T, gx, s_jmp, s_acc, s_cnt, s_msk, dep, cl, msk);
    if (!ok) {
      if (tid == 0) report(a.dev_err, TL_EBADTREE);
      wait_vmem();   // let the in-flight LDS copies land before the block retires
      return;
    }
    __syncthreads();   // topology scratch is dead from here
    if (tid < T) {
      s_cl[tid] = cl * kLog2e;
      s_beta[tid] = bx;
      const int I = tid / kTile;
#pragma unroll
      for (int w = 0; w < W; ++w) {
        s_mask[tid * W + w] = msk[w];
        if (msk[w]) atomicOr(reinterpret_cast<unsigned long long*>(&s_tmask[I * W + w]),
                             (unsigned long long)msk[w]);
      }
      // strict ancestors of this node inside its own tile
      uint64_t wv = msk[0];
#pragma unroll
      for (int w = 1; w < W; ++w)
        if ((tid >> 6) == w) wv = msk[w];
      const uint32_t in_tile = (uint32_t)(wv >> ((I & 3) * kTile)) & 0xFFFFu & ~(1u << (tid & 15));
      if (in_tile) atomicOr(&s_tin[I], in_tile);
    }
  }
  wait_vmem();
  __syncthreads();   // K, U^T, masks and decays are in LDS
  TL_TRACE_POINT(a, 3);

  // the wave's state rows, split into bf16 hi + lo MFMA A operands
  bf16x8 shi[KS], slo[KS];
  if (vw) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) split8_bf16(sraw[ks][0], sraw[ks][1], shi[ks], slo[ks]);
  }

  // operand fragment of row R + lr of the swizzled K rows (R a multiple of 16)
  const int key = lr & (CPRK - 1);
  const int fo_row = lr * D * 2;
  const unsigned char* kbase = reinterpret_cast<const unsigned char*>(s_k);
  auto kfrag = [&](int R, int ks) {
    const unsigned char* p = kbase + R * D * 2 + fo_row;
    return *reinterpret_cast<const bf16x8*>(p + (((4 * ks + lg) ^ key) * 16));
  };
  // A-operand fragment of U^T row (16 w + lr), node chunk c
  const int uo = ((kTile * wave + lr) * TS + 4 * lg) * 2;
  auto ufrag = [&](const __bf16* base, int c) {
    const unsigned char* p = reinterpret_cast<const unsigned char*>(base) + uo + 64 * c;
    const bf16x4 x0 = *reinterpret_cast<const bf16x4*>(p);
    const bf16x4 x1 = *reinterpret_cast<const bf16x4*>(p + 32);
    return bf16x8{x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
  };
  // chunk operands: [chunk][piece][lane] 16 bytes, pieces C hi, C lo, -G hi, -G lo

  // ---- node tiles
  const int nt = (T + kTile - 1) / kTile;
  float* obase = a.out + (size_t)off * v_row + (size_t)h * D + kTile * wave + 4 * lg;

  // Q fragments (B operand, columns = nodes of tile I) and V rows of tile I,
  // loaded unconditionally from rows clamped to T - 1: columns >= T only
  // reach masked coefficients or outputs that are never stored, and fixed
  // load counts let the compiler wait for exactly the loads it needs
  auto load_q = [&](int I, bf16x8 (&dst)[KS]) {
    const int r = min(kTile * I + lr, T - 1);
    const __bf16* row = Qb + (size_t)r * qk_row;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      dst[ks] = *reinterpret_cast<const bf16x8*>(row + ks * 32 + 8 * lg);
    }
  };
  auto load_v = [&](int I) {
    const int r = min(kTile * I + lr, T - 1);
    const int col = min(kTile * wave, D - kTile) + 4 * lg;   // waves without value rows read a valid column
    return *reinterpret_cast<const bf16x4*>(Vb + (size_t)r * v_row + col);
  };

  // per-tile values of this lane's node (column i = 16 I + lr); the mask
  // words are read from LDS where needed (a register array indexed by a
  // runtime word number would live in scratch)
  struct TileIn {
    float cli, bi;
  };
  auto tile_in = [&](int I, TileIn& t) __attribute__((always_inline)) {
    const int i = kTile * I + lr;
    const bool iv = i < T;
    const float cv = s_cl[i];
    t.cli = iv ? cv : 0.f;
    const float bv = s_beta[min(i, tm - 1)];
    t.bi = iv ? bv : 0.f;
  };
  // 32 bits of tile I's OR mask starting at node 32 c (uniform)
  auto tile_bits32 = [&](int I, int c) __attribute__((always_inline)) {
    return (unsigned)(s_tmask[I * W + (c >> 1)] >> ((c & 1) * 32));
  };

  // 1. coefficient chunks of tile I, shared over the waves, into buffer buf.
  // The work is dealt out by half-chunk (one 16-node tile J each), so that a
  // wave carries at most one half-chunk per node tile (NW >= 8 at d = 128).
  auto chunks = [&](int I, const bf16x8 (&qf)[KS], const TileIn& t, unsigned char* buf, float* gin)
                    __attribute__((always_inline)) {
    const int nh = 2 * (I / 2 + 1);   // tiles 0 .. 2 (I / 2) + 1: whole chunks
    const int i = kTile * I + lr;
    for (int J = wave; J < nh; J += NW) {   // uniform
      const int c = J >> 1, hf = J & 1;
      const unsigned bits = (tile_bits32(I, c) >> (hf * kTile)) & 0xFFFFu;
      float cv[4] = {0.f, 0.f, 0.f, 0.f}, gv[4] = {0.f, 0.f, 0.f, 0.f};
      if (J <= I && bits) {   // uniform
        bf16x8 kj[KS], kfi[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          kj[ks] = kfrag(kTile * J, ks);
          kfi[ks] = kfrag(kTile * I, ks);
        }
        const uint64_t mw = (i < T) ? s_mask[i * W + (J >> 2)] : 0ull;   // M+ row of node i
        const f32x4 clj = *reinterpret_cast<const f32x4*>(s_cl + kTile * J + 4 * lg);
        f32x4 qk = f32x4{0.f, 0.f, 0.f, 0.f}, kk = qk;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          qk = mfma16(kj[ks], qf[ks], qk);               // rows j, column i: k_j . q_i
          kk = mfma16(kj[ks], kfi[ks], kk);
        }
        const unsigned mb = (unsigned)(mw >> ((J & 3) * kTile + 4 * lg)) & 0xFu;
        const unsigned self = (J == I) ? (1u << lr) >> (4 * lg) : 0u;   // bit r: j == i
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const bool m = (mb >> r) & 1u;
          const float dec = __builtin_amdgcn_exp2f(t.cli - clj[r]);
          cv[r] = m ? (dec * a.q_scale) * qk[r] : 0.f;
          gv[r] = (m && !((self >> r) & 1u)) ? (t.bi * dec) * kk[r] : 0.f;
        }
      }
      if (J == I) {   // the in-tile block: row-major to LDS, zero in the operand
        *reinterpret_cast<f32x4*>(gin + lr * kTile + 4 * lg) = f32x4{gv[0], gv[1], gv[2], gv[3]};
#pragma unroll
        for (int r = 0; r < 4; ++r) gv[r] = 0.f;
      }
      // this half's 8 bytes of each 16-byte operand piece: hi01 hi23, then lo01 lo23
      uint32_t cw[4], gw[4];
      split2_bf16(cv[0], cv[1], cw[0], cw[2]);
      split2_bf16(cv[2], cv[3], cw[1], cw[3]);
      unsigned char* pc = buf + ((c * NF) * 64 + lane) * 16 + hf * 8;
      *reinterpret_cast<uint2*>(pc) = uint2{cw[0], cw[1]};
      *reinterpret_cast<uint2*>(pc + 1024) = uint2{cw[2], cw[3]};
      // G stored negated: U^T (-G)^T is subtracted by accumulation
      split2_bf16(-gv[0], -gv[1], gw[0], gw[2]);
      split2_bf16(-gv[2], -gv[3], gw[1], gw[3]);
      *reinterpret_cast<uint2*>(pc + 2048) = uint2{gw[0], gw[1]};
      *reinterpret_cast<uint2*>(pc + 3072) = uint2{gw[2], gw[3]};
    }
  };

  // 2.-3. value rows of this wave for tile I: the delta-rule solve, then the
  // readout; returns O^T (the store is left to the caller).  The chunks of
  // earlier tiles hold final U^T columns, so their correction and readout
  // terms run as interleaved MFMA chains, independent of the B0 products;
  // only the chunk of tile I itself waits for the in-tile solve.
  struct ChunkOps {
    bf16x8 ch, cl, gh, gl, uh, ul;
  };
  // U^T of every completed chunk (both of its tiles solved), this wave's
  // rows, kept in registers once read back
  constexpr int NCU = 2 * W;
  bf16x8 ureg_h[NCU], ureg_l[NCU];
  auto value_work = [&](int I, const bf16x8 (&qf)[KS], const bf16x4 vcur, const TileIn& t,
                        const unsigned char* buf, const float* gin) __attribute__((always_inline)) {
    const int cI = I / 2;   // the chunk that holds tile I
    const int i = kTile * I + lr;
    const bool iv = i < T;
    auto pc = [&](int c, int k) __attribute__((always_inline)) { return buf + ((c * NF + k) * 64 + lane) * 16; };
    auto load_ops = [&](int c, ChunkOps& o) __attribute__((always_inline)) {
      o.ch = *reinterpret_cast<const bf16x8*>(pc(c, 0));
      o.cl = *reinterpret_cast<const bf16x8*>(pc(c, 1));
      o.uh = ufrag(s_ut, c);
      o.gh = *reinterpret_cast<const bf16x8*>(pc(c, 2));
      o.gl = *reinterpret_cast<const bf16x8*>(pc(c, 3));
      o.ul = ufrag(s_utl, c);
    };
    // chunks with an ancestor of tile I (uniform)
    uint32_t live = 0;
#pragma unroll
    for (int c = 0; c < 2 * W; ++c) live |= (tile_bits32(I, c) != 0u ? 1u : 0u) << c;
    live = __builtin_amdgcn_readfirstlane(live);
    f32x4 x = f32x4{0.f, 0.f, 0.f, 0.f}, acc = x, acc2 = x;
    // B0^T = S Q_I^T and S K_I^T, independent of the chunks
    f32x4 b0 = f32x4{0.f, 0.f, 0.f, 0.f}, sk = b0;
    bf16x8 kfi[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) kfi[ks] = kfrag(kTile * I, ks);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      b0 = mfma16(shi[ks], qf[ks], b0);
      b0 = mfma16(slo[ks], qf[ks], b0);
      sk = mfma16(shi[ks], kfi[ks], sk);
      sk = mfma16(slo[ks], kfi[ks], sk);
    }
    // the chunks of earlier tiles
    {
#pragma unroll
      for (int c = 0; c < NCU; ++c) {   // completed chunks: U^T from registers
        if (c >= cI || !((live >> c) & 1u)) continue;   // uniform
        ChunkOps o;
        o.ch = *reinterpret_cast<const bf16x8*>(pc(c, 0));
        o.cl = *reinterpret_cast<const bf16x8*>(pc(c, 1));
        o.gh = *reinterpret_cast<const bf16x8*>(pc(c, 2));
        o.gl = *reinterpret_cast<const bf16x8*>(pc(c, 3));
        o.uh = ureg_h[c];
        o.ul = ureg_l[c];
        x = mfma16(o.uh, o.gh, x);
        acc = mfma16(o.uh, o.ch, acc);
        x = mfma16(o.uh, o.gl, x);
        acc2 = mfma16(o.uh, o.cl, acc2);
        x = mfma16(o.ul, o.gh, x);
        acc = mfma16(o.ul, o.ch, acc);
      }
    }
    const float Pi = iv ? __builtin_amdgcn_exp2f(t.cli) : 0.f;

    {
      // 2. U_I: X = beta (V - P S K^T) - U^T G^T over the earlier tiles (in x),
      // then the chunk of tile I: the G columns of tile I are zero there (its
      // block is solved below) and those of tile I - 1 are final
      ChunkOps o;
      load_ops(cI, o);
      x = mfma16(o.uh, o.gh, x);
      x = mfma16(o.uh, o.gl, x);
      x = mfma16(o.ul, o.gh, x);
#pragma unroll
      for (int r = 0; r < 4; ++r) x[r] += t.bi * ((float)vcur[r] - Pi * sk[r]);
      // ... then the in-tile ancestors, in index order (lane (j, lg) holds u_j)
      // (lane j of each 16-lane row broadcast to its row by DPP row_newbcast)
      const unsigned tin = s_tin[I];
      auto step = [&](auto jc) __attribute__((always_inline)) {
        constexpr int j = decltype(jc)::value;
        if ((tin >> j) & 1u) {   // uniform
          const float gij = gin[lr * kTile + j];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float uj = __int_as_float(
                __builtin_amdgcn_update_dpp(0, __float_as_int(x[r]), 0x150 + j, 0xF, 0xF, false));
            x[r] -= gij * uj;
          }
        }
      };
      static_for<kTile>(step);
      // U_I^T -> LDS as bf16 hi + lo (zero for nodes >= T)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float uval = iv ? x[r] : 0.f;
        const uint32_t ub = __float_as_uint(uval);
        const float rem = uval - __uint_as_float(ub & 0xffff0000u);
        const int at = (kTile * wave + 4 * lg + r) * TS + i;
        s_ut[at] = __builtin_bit_cast(__bf16, (uint16_t)(ub >> 16));
        s_utl[at] = (__bf16)rem;
      }
      // 3. the readout term of tile I's chunk, with U_I now in place (the
      // wave's own rows: its LDS writes above are read back in order)
      const bf16x8 uh = ufrag(s_ut, cI), ul = ufrag(s_utl, cI);
      acc = mfma16(uh, o.ch, acc);
      acc2 = mfma16(uh, o.cl, acc2);
      acc = mfma16(ul, o.ch, acc);
      // chunk cI is complete after an odd tile: keep its U^T.  Every entry
      // is rewritten (a select), so the array is only ever indexed statically
      const bool done = (I & 1) != 0;
#pragma unroll
      for (int c = 0; c < NCU; ++c) {
        const bool here = done && c == cI;
        ureg_h[c] = here ? uh : ureg_h[c];
        ureg_l[c] = here ? ul : ureg_l[c];
      }
    }
    // 3. O^T = q_scale P_i B0^T + U^T C^T
    const float ps = Pi * a.q_scale;
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[r] = ps * b0[r] + (acc[r] + acc2[r]);
    return acc;
  };

  // tile I's chunk operands: buffer I & 1 when double-buffered, else the only one
  auto bufp = [&](int I) { return (DB && (I & 1)) ? tl_lds + L.frag2 : s_frag; };
  auto ginp = [&](int I) { return s_gin + (DB ? (I & 1) * kTile * kTile : 0); };

  // Pipeline.  Double-buffered: step I forms the chunks of tile I + 1 (buffer
  // (I + 1) & 1, free since the previous barrier) while the value work of
  // tile I reads buffer I & 1, so one barrier per tile.  Single buffer: value
  // work, barrier, chunks of the next tile, barrier.  Q rows are prefetched
  // two tiles ahead into three register buffers that change roles from step
  // to step (the tile loop is unrolled three times).  Each tile's output is
  // stored in the next step, next to that step's prefetch.
  bf16x8 q0[KS], q1[KS], q2[KS];   // Q fragments of tiles I, I + 1, I + 2
  bf16x4 v0 = load_v(0), v1 = load_v(1);
  load_q(0, q0);
  load_q(1, q1);
  {
    TileIn t;
    tile_in(0, t);
    chunks(0, q0, t, bufp(0), ginp(0));
  }
  lds_barrier();
  TL_TRACE_POINT(a, 4);

  f32x4 pend = f32x4{0.f, 0.f, 0.f, 0.f};
  int pend_row = -1;
  // one node tile: qa / va hold tile I, qb / vb tile I + 1, qc / vc receive
  // tile I + 2; the three buffers change roles from tile to tile, so no
  // prefetched register is copied (a copy would wait for its load)
  auto tile_step = [&](int I, bf16x8 (&qa)[KS], bf16x8 (&qb)[KS], bf16x8 (&qc)[KS], bf16x4& va,
                       [[maybe_unused]] bf16x4& vb, bf16x4& vc) __attribute__((always_inline)) {
    // Forming the chunks of tile I + 1 consumes its Q rows, and that wait
    // covers every load and store issued before it (one counter, which the
    // compiler drains when both are pending).  So the output store and the
    // prefetch of tile I + 2 are issued after it: the next step's wait then
    // covers only work issued a whole step earlier.
    if (DB && I + 1 < nt) {
      TileIn tn;
      tile_in(I + 1, tn);
      chunks(I + 1, qb, tn, bufp(I + 1), ginp(I + 1));
    }
    if (vw && pend_row >= 0) store_out<true>(obase + (size_t)pend_row * v_row, pend);
    pend_row = -1;
    load_q(I + 2, qc);   // rows clamped: harmless past the last tile
    vc = load_v(I + 2);
    if (vw) {
      TileIn t;
      tile_in(I, t);
      pend = value_work(I, qa, va, t, bufp(I), ginp(I));
      if (kTile * I + lr < T) pend_row = kTile * I + lr;
    }
    if constexpr (DB) {
      lds_barrier();   // chunks of tile I + 1 visible; buffer I & 1 free again
    } else if (I + 1 < nt) {
      lds_barrier();   // every wave is done with the chunk buffer
      TileIn tn;
      tile_in(I + 1, tn);
      chunks(I + 1, qb, tn, bufp(I + 1), ginp(I + 1));
      lds_barrier();   // chunks of tile I + 1 are in LDS
    }
    if (I < 2) TL_TRACE_POINT(a, 5 + I);
  };
  bf16x4 v2 = bf16x4{};
  for (int I = 0; I < nt; I += 3) {   // uniform
    tile_step(I, q0, q1, q2, v0, v1, v2);
    if (I + 1 < nt) tile_step(I + 1, q1, q2, q0, v1, v2, v0);
    if (I + 2 < nt) tile_step(I + 2, q2, q0, q1, v2, v0, v1);
  }
  if (vw && pend_row >= 0) store_out<true>(obase + (size_t)pend_row * v_row, pend);
  TL_TRACE_POINT(a, 15);
}

// LDS bytes of the tiled kernel for a node cap (double-buffered if that fits).
int verify_tiled_lds_bytes(int d, int tm, int W) {
  const int db = tiled_layout(d, tm, W, true).total;
  return db <= 160 * 1024 ? db : tiled_layout(d, tm, W, false).total;
}

template <int D, int W, bool DB>
static tl_status launch_tiled_one(const VerifyArgs& a, hipStream_t stream) {
  const int lds = tiled_layout(D, a.tm, W, DB).total;
  if (lds > 160 * 1024) return TL_EUNSUPPORTED;
  const long blocks = 8 * (((long)a.batch * a.Hk + 7) / 8) * (a.Hv / a.Hk);
  if (blocks == 0) return TL_OK;
  if (blocks > 0x7fffffffL) return TL_EINVAL;
  auto kern = verify_tiled_kernel<D, W, DB>;
  if (lds > 64 * 1024) {
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                            hipFuncAttributeMaxDynamicSharedMemorySize, lds) != hipSuccess)
      return TL_EHIP;
  }
  VerifyArgs b = a;
  b.lds_bytes = lds;
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(64 * tiled_waves(D)), lds, stream, b);
  return hipGetLastError() == hipSuccess ? TL_OK : TL_EHIP;
}

template <int D, int W>
static tl_status launch_tiled_db(const VerifyArgs& a, hipStream_t stream) {
  if (tiled_layout(D, a.tm, W, true).total <= 160 * 1024) return launch_tiled_one<D, W, true>(a, stream);
  return launch_tiled_one<D, W, false>(a, stream);
}

template <int D>
static tl_status launch_tiled_w(const VerifyArgs& a, hipStream_t stream) {
  if (a.tm > 128) return launch_tiled_db<D, 4>(a, stream);
  if (a.tm > 64) return launch_tiled_db<D, 2>(a, stream);
  return launch_tiled_db<D, 1>(a, stream);
}

tl_status launch_verify_tiled(const tl_problem& p, const VerifyArgs& a, hipStream_t stream) {
  if (p.mode != TL_MODE_GDN) return TL_EUNSUPPORTED;
  switch (p.d_k) {
    case 32: return launch_tiled_w<32>(a, stream);
    case 64: return launch_tiled_w<64>(a, stream);
    case 128: return launch_tiled_w<128>(a, stream);
    default: return TL_EUNSUPPORTED;
  }
}

}  // namespace tl
