// Verify, gated delta rule on MFMA, trees of up to 128 nodes at d = 128:
// the correction system solved once per workgroup as an explicit inverse,
// so that the value work is a few dense products with no chain over node
// tiles.
//
// Theorem 1 (§4.1) with Lemma 2 for the delta rule, per (request, v-head):
//   R = D_beta (V - D_P K S^T)                 R_j = beta_j (v_j - P_j S k_j)
//   G_ij = beta_i 2^(cl_i - cl_j) (k_i . k_j)  for strict ancestors j of i
//   U = (I + G)^{-1} R                         (Lemma 3: I + G is unit lower
//                                              triangular in index order)
//   O = q_scale (D_P Q S^T + C U)              C_ij = [j in Anc(i) u {i}]
//                                                     2^(cl_i - cl_j) (q_i . k_j)
// (stored orientation: S is the [d_v, d_k] slot; cl is the cumulative log2
// decay along the root path.)
//
// The node-by-node coupling sits in A = (I + G)^{-1}, a T x T matrix that does
// not depend on the value channels.  So one workgroup of 8 wave64s per
// (request, v-head) runs three phases separated by two barriers, after a
// prologue in which wave 0 forms the topology alone (wave_topology_jump, no
// workgroup barrier) while waves 1..7 issue the K, Q and V copies:
//  1. every wave forms its share of the 16 x 16 blocks (I, J <= I) of C and G
//     (K_J Q_I^T and K_J K_I^T on MFMA, masked by the M+ rows, decayed) into
//     LDS in MFMA operand order, and of the in-tile inverses (I + G_II)^{-1}
//     (forward substitution on the identity, each step broadcasting a column
//     of the tile along its 16-lane row by DPP); then, for its own 16 value
//     channels, B0 = Q S^T and SK = K S^T over all node tiles (state in bf16
//     hi + lo) and R from SK;
//  2. wave J forms column block J of A: for I = J, J + 1, ...,
//       X_I = (I + G_II)^{-1} (delta_IJ - sum_{J <= K < I} G_IK X_K),
//     all on MFMA: X_K come out of the products as the B operands of the
//     next ones, and so does column block J of C A, (C A)_IJ =
//     sum_{J <= K <= I} C_IK X_K.  Columns are independent, so the waves
//     need no barrier between them.  C A goes to LDS over the dead Q and K
//     rows (A itself is never stored);
//  3. every wave forms O = q_scale P B0 + (C A) R for its value channels
//     (C U = C (A R)): products of an LDS operand (C A) with the register
//     fragments of R, no LDS round trip for the value side.
// Blocks of C, G, A and C A whose tile pair holds no ancestor relation are
// zero and are neither formed nor read.  The matrices are fp32, split into bf16
// hi + lo for the MFMA, with fp32 accumulation.
#include <hip/hip_runtime.h>

#include <utility>

#include "tl_device.h"
#include "tl_kernels.h"
#include "verify_common.h"

namespace tl {

namespace {

constexpr int kDenseWaves = 8;                     // one per 16 value channels (d = 128)
constexpr int kDenseThreads = 64 * kDenseWaves;
constexpr int kDenseMaxTiles = 8;   // 128 nodes

// MFMA 16x16x16 bf16: D = A (16 x 16) * B (16 x 16) + C.  Lane l supplies A
// row (l % 16) and B column (l % 16), 4 values each of the K range owned by
// lane group l / 16; D comes back as rows 4 (l / 16) .. + 3 of column l % 16.
// So a D fragment is directly the B operand of a product whose K index is
// D's row index.
__device__ inline f32x4 mfma16k(const bf16x4& a, const bf16x4& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4, a),
                                                   __builtin_bit_cast(s16x4, b), c, 0, 0, 0);
}

// f32x4 -> bf16x4 hi + lo (split2_bf16 on both pairs)
__device__ inline void split4_bf16(const f32x4& x, bf16x4& hi, bf16x4& lo) {
  uint32_t h0, h1, l0, l1;
  split2_bf16(x[0], x[1], h0, l0);
  split2_bf16(x[2], x[3], h1, l1);
  hi = __builtin_bit_cast(bf16x4, uint2{h0, h1});
  lo = __builtin_bit_cast(bf16x4, uint2{l0, l1});
}

__host__ __device__ constexpr int tri(int n) { return n * (n + 1) / 2; }

// Blocks are stored in pairs of node tiles (J0, J0 + 1), J0 even, so that one
// 16-byte read per lane yields a whole 16x16x32 operand: a 1 KB plane of
// hi parts, [lane][hi of J0 | hi of J0 + 1], then one of lo parts, 2 KB a
// pair (16 bytes per lane per plane, so the reads are free of bank
// conflicts).
// Row I of a lower-triangular set (J <= I) holds I / 2 + 1 pairs (the half
// J = I + 1 of an even row is kept zero); pair_row(I) is its first pair.
// The strictly lower set of G (K < I) holds (I + 1) / 2 pairs a row.
__host__ __device__ constexpr int pair_row(int I) { return (I / 2) * (I / 2 + 1) + ((I & 1) ? I / 2 + 1 : 0); }
__host__ __device__ constexpr int gpair_row(int I) { return (I / 2) * (I / 2) + ((I & 1) ? I / 2 : 0); }

}  // namespace

struct DenseLayout {
  int flag, cl, beta, mask, tmask, tin, gin, kq, cst, gst, ainv, total;
};

// LDS layout (bytes); identical on host and device.
__host__ __device__ inline DenseLayout dense_layout(int tm, int W) {
  const int nb = tm / kTile;
  DenseLayout L;
  int o = 0;
  L.flag = o;  o += 16;                              // the tree is malformed
  L.cl = o;    o += align16((tm + 16) * 4);          // cumulative log2-decay
  L.beta = o;  o += align16(tm * 4);
  L.mask = o;  o += tm * W * 8;                      // M+ rows
  L.tmask = o; o += align16(nb * W * 8);             // OR of M+ rows per node tile
  L.tin = o;   o += align16(nb * 4);                 // in-tile strict ancestors per tile
  L.gin = o;   o += nb * kTile * kTile * 4;          // in-tile blocks of G, row-major fp32
  L.kq = o;                                          // K and Q rows | the blocks of C A
  {
    const int rows = 2 * tm * 128 * 2, ablk = pair_row(nb) * 2048;
    o += rows > ablk ? rows : ablk;
  }
  L.cst = o;                                         // blocks of C | staged V rows
  {
    const int cb = pair_row(nb) * 2048, vb = tm * 128 * 2;
    o += cb > vb ? cb : vb;
  }
  L.gst = o;                                         // strictly lower blocks of -G | topology scratch
  {
    const int gb = gpair_row(nb) * 2048, topo = kThreads * (4 + 4 + 4) + kThreads * W * 8;
    o += gb > topo ? gb : topo;
  }
  L.ainv = o;  o += nb * 1024;                      // (I + G_II)^-1 per node tile, bf16 hi | lo
  L.total = o;
  return L;
}

template <int W>
// One workgroup per CU (LDS), so two waves per SIMD: the compiler may spend
// the registers that allows on overlapping LDS reads with products.
__global__ __launch_bounds__(kDenseThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void verify_gdn_dense_kernel(VerifyArgs a) {
  constexpr int D = 128;
  constexpr int KS = D / 32;
  constexpr int CPRK = D / 8;
  constexpr int NTM = kDenseMaxTiles;
  constexpr float kLog2e = 1.4426950408889634f;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, lr = lane & 15, lg = lane >> 4;
  lds_poison(a.lds_bytes);
  TL_TRACE_POINT(a, 0);
#ifdef TL_TRACE
  if (a.trace && threadIdx.x == 0) a.trace[(size_t)blockIdx.x * 16 + 13] = (long long)__builtin_readcyclecounter();
#endif

  // ---- block -> (request, qk-head, v-head): grouped v-heads 8 ids apart (same XCD)
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
  const int nt = (T + kTile - 1) / kTile;   // node tiles of this tree (uniform)
  const DenseLayout L = dense_layout(tm, W);
  float* s_cl = reinterpret_cast<float*>(tl_lds + L.cl);
  float* s_beta = reinterpret_cast<float*>(tl_lds + L.beta);
  uint64_t* s_mask = reinterpret_cast<uint64_t*>(tl_lds + L.mask);
  uint64_t* s_tmask = reinterpret_cast<uint64_t*>(tl_lds + L.tmask);
  uint32_t* s_tin = reinterpret_cast<uint32_t*>(tl_lds + L.tin);
  float* s_gin = reinterpret_cast<float*>(tl_lds + L.gin);
  __bf16* s_k = reinterpret_cast<__bf16*>(tl_lds + L.kq);
  __bf16* s_q = s_k + tm * D;
  unsigned char* s_a = tl_lds + L.kq;      // blocks of C A, over the dead K and Q rows
  unsigned char* s_c = tl_lds + L.cst;
  __bf16* s_v = reinterpret_cast<__bf16*>(s_c);   // staged V rows, until the blocks of C are formed
  unsigned char* s_g = tl_lds + L.gst;
  unsigned char* s_ainv = tl_lds + L.ainv;   // in-tile inverses, A operands of 16x16x16 products

  const size_t qk_row = (size_t)a.Hk * D, v_row = (size_t)a.Hv * D;
  const __bf16* Qb = reinterpret_cast<const __bf16*>(a.q) + (size_t)off * qk_row + (size_t)hq * D;
  const __bf16* Kb = reinterpret_cast<const __bf16*>(a.k) + (size_t)off * qk_row + (size_t)hq * D;
  const __bf16* Vb = reinterpret_cast<const __bf16*>(a.v) + (size_t)off * v_row + (size_t)h * D;

  // ---- prologue.  Wave 0 loads the parents and gates and forms the
  // topology alone (no workgroup barrier) while waves 1..7 issue the direct
  // copies of the K, Q and V rows into swizzled LDS; every wave then loads
  // its state rows (needed last, in phase 1b).  The copies are issued as
  // inline assembly, which the compiler does not count, and loads complete
  // in issue order.
  TL_TRACE_POINT(a, 1);
  // The parents, gates and copies are issued at raised wave priority and the
  // state rows at the normal one, so that every wave's copies reach the
  // memory queue before any wave's state rows (the older waves would
  // otherwise win the issue arbitration with their state loads).
  __builtin_amdgcn_s_setprio(2);
  constexpr int NE = W;   // nodes per lane of wave 0 (node cap <= 64 W)
  int par[NE];
  float gx[NE], bx[NE];
  if (wave == 0) {   // uniform
#pragma unroll
    for (int e = 0; e < NE; ++e) {   // unconditional loads, clamped to the tree
      const int i = off + min(lane + 64 * e, T - 1);
      par[e] = a.parent[i];
      gx[e] = a.g[(size_t)i * a.Hv + h];
      bx[e] = a.beta[(size_t)i * a.Hv + h];
    }
  }
  // the parents and gates enter this CU's memory queue ahead of the bulk
  // copies (a barrier without a memory wait: wave 0's loads are issued, not
  // complete)
  __builtin_amdgcn_s_barrier();
  if (wave > 0) {   // uniform
    constexpr int CT = kDenseThreads - 64;
    for (int base = (wave - 1) * 64; base < T * CPRK; base += CT) {
      const int p = base + lane;
      if (p < T * CPRK) {
        const int r = p / CPRK, c = swz<CPRK>(r, p % CPRK);
        copy16_to_lds_async(Kb + (size_t)r * qk_row + c * 8, s_k + (size_t)base * 8);
        copy16_to_lds_async(Qb + (size_t)r * qk_row + c * 8, s_q + (size_t)base * 8);
      }
    }
    // the V rows of every node tile, into the C region (rows past T repeat
    // row T - 1; their R entries are set to zero)
    for (int base = (wave - 1) * 64; base < kTile * nt * CPRK; base += CT) {
      const int p = base + lane, r = p / CPRK, c = swz<CPRK>(r, p % CPRK);
      if (p < kTile * nt * CPRK)
        copy16_to_lds_async(Vb + (size_t)min(r, T - 1) * v_row + c * 8, s_v + (size_t)base * 8);
    }
  }
  TL_TRACE_POINT(a, 6);
  // S^T as the B operand of 16x16x32 products: column = channel 16 wave + lr
  // (a row of the stored slot), K = key channels 32 ks + 8 lg .. + 7 of chunk
  // ks for lane group lg (the products over d_k take K in this order, so a K
  // or Q operand is one 16-byte chunk of a staged row)
  f32x4 sraw[KS][2];
  __builtin_amdgcn_s_setprio(0);
  {
    const float* row = a.state + ((size_t)sidx * a.Hv + h) * D * D + (size_t)(kTile * wave + lr) * D;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      sraw[ks][0] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(row + ks * 32 + 8 * lg));
      sraw[ks][1] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(row + ks * 32 + 8 * lg + 4));
    }
  }

  // ---- topology, by wave 0: M+ rows, cumulative log-decay, per-tile masks
  TL_TRACE_POINT(a, 2);
  int* s_flag = reinterpret_cast<int*>(tl_lds + L.flag);
  if (wave == 0) {   // uniform
    for (int x = lane; x < (tm / kTile) * W; x += 64) s_tmask[x] = 0;
    for (int x = lane; x < tm / kTile; x += 64) s_tin[x] = 0u;
    int* s_jmp = reinterpret_cast<int*>(s_g);
    float* s_acc = reinterpret_cast<float*>(s_jmp + 64 * NE);
    uint64_t* s_msk = reinterpret_cast<uint64_t*>(s_acc + 64 * NE);
    float cl[NE];
    uint64_t msk[NE][W];
    const bool ok = wave_topology_jump<W, NE>(par, gx, T, s_jmp, s_acc, s_msk, cl, msk);
    if (lane == 0) {
      *s_flag = ok ? 0 : 1;
      if (!ok) report(a.dev_err, TL_EBADTREE);
    }
    if (ok) {   // uniform
#pragma unroll
      for (int e = 0; e < NE; ++e) {
        const int i = lane + 64 * e;
        if (i < T) {
          s_cl[i] = cl[e] * kLog2e;
          s_beta[i] = bx[e];
          const int I = i / kTile;
#pragma unroll
          for (int w = 0; w < W; ++w) {
            s_mask[i * W + w] = msk[e][w];
            if (msk[e][w]) atomicOr(reinterpret_cast<unsigned long long*>(&s_tmask[I * W + w]),
                                    (unsigned long long)msk[e][w]);
          }
          // node i's ancestors inside its tile: bits (I % 4) 16 .. + 15 of word e
          const uint32_t in_tile = (uint32_t)(msk[e][e] >> ((I & 3) * kTile)) & 0xFFFFu & ~(1u << (i & 15));
          if (in_tile) atomicOr(&s_tin[I], in_tile);
        }
      }
    }
  }
  TL_TRACE_POINT(a, 7);
  // the K, Q and V copies (issued before the state loads) have landed once
  // at most the state loads of this wave are outstanding
  wait_vmem_below<2 * KS>();
  lds_barrier();   // K, Q, V, masks and decays are in LDS (the state stays in flight)
  if (*s_flag) {   // uniform: a malformed tree (reported by wave 0)
    wait_vmem();   // the state rows land before the block retires
    return;
  }
  // V[node 16 J + 4 lg + e][channel 16 wave + lr] by LDS transpose reads: lane
  // (lg, lr) names row 16 J + 4 lg + lr / 4 and channels 16 wave + 4 (lr % 4)
  // .. + 3, so it receives channel 16 wave + lr of nodes 16 J + 4 lg .. + 3
  bf16x4 vv[NTM];
  {
    const int vrow_l = 4 * lg + (lr >> 2);
    const int col = kTile * wave + 4 * (lr & 3);
    const int vo = vrow_l * D * 2 + swz<CPRK>(vrow_l, col >> 3) * 16 + (col & 7) * 2;
#pragma unroll
    for (int J = 0; J < NTM; ++J)   // rows 16 J + vrow_l keep the swizzle key of row vrow_l
      vv[J] = J < nt ? lds_read_tr16(s_v, vo + (kTile * J) * D * 2) : bf16x4{};
  }
  lds_barrier();   // every wave has read the staged V rows (the C blocks go over them)
  TL_TRACE_POINT(a, 3);

  // operand fragment of row R + lr of the swizzled K or Q rows (R a multiple
  // of 16): key channels 32 ks + 8 lg .. + 7, i.e. 16-byte chunk 4 ks + lg of
  // the row, one read (the swizzle puts the 16 rows' chunks on distinct banks)
  const int key = lr & (CPRK - 1);
  const int fo_row = lr * D * 2;
  auto frag = [&](const __bf16* base, int R, int ks) __attribute__((always_inline)) {
    const unsigned char* p = reinterpret_cast<const unsigned char*>(base) + R * D * 2 + fo_row;
    return *reinterpret_cast<const bf16x8*>(p + (((4 * ks + lg) ^ key) * 16));
  };
  // block x (fp32, MFMA fragment layout) into half `half` of pair `pair`
  auto put_half = [&](unsigned char* base, int pair, int half, const f32x4& x) __attribute__((always_inline)) {
    bf16x4 hi, lo;
    split4_bf16(x, hi, lo);
    unsigned char* q = base + pair * 2048 + lane * 16 + half * 8;
    *reinterpret_cast<bf16x4*>(q) = hi;
    *reinterpret_cast<bf16x4*>(q + 1024) = lo;
  };
  auto zero_half = [&](unsigned char* base, int pair, int half) __attribute__((always_inline)) {
    unsigned char* q = base + pair * 2048 + lane * 16 + half * 8;
    *reinterpret_cast<uint2*>(q) = uint2{0u, 0u};
    *reinterpret_cast<uint2*>(q + 1024) = uint2{0u, 0u};
  };
  auto get_pair = [&](const unsigned char* base, int pair, bf16x8& hi, bf16x8& lo) __attribute__((always_inline)) {
    const unsigned char* q = base + pair * 2048 + lane * 16;
    hi = *reinterpret_cast<const bf16x8*>(q);
    lo = *reinterpret_cast<const bf16x8*>(q + 1024);
  };
  // fp32 fragment x -> half `half` of a register pair operand (hi, lo)
  // (`half` is a compile-time constant wherever this is used)
  auto set_half = [&](bf16x8& hi, bf16x8& lo, int half, const f32x4& x) __attribute__((always_inline)) {
    bf16x4 h, l;
    split4_bf16(x, h, l);
    if (half == 0) {
      hi = bf16x8{h[0], h[1], h[2], h[3], hi[4], hi[5], hi[6], hi[7]};
      lo = bf16x8{l[0], l[1], l[2], l[3], lo[4], lo[5], lo[6], lo[7]};
    } else {
      hi = bf16x8{hi[0], hi[1], hi[2], hi[3], h[0], h[1], h[2], h[3]};
      lo = bf16x8{lo[0], lo[1], lo[2], lo[3], l[0], l[1], l[2], l[3]};
    }
  };

  // tile pairs (I, J <= I) that hold an ancestor relation, as one uniform
  // 64-bit mask (bit 8 I + J); other blocks of C, G and A are zero
  uint64_t live_bits;
  {
    const int I = lane >> 3, J = lane & 7;   // lane 8 I + J tests tile pair (I, J)
    const uint64_t m = s_tmask[min(I, tm / kTile - 1) * W + min(J >> 2, W - 1)];
    live_bits = __ballot(J <= I && I < nt && ((m >> ((J & 3) * kTile)) & 0xFFFFull) != 0ull);
  }
  auto live = [&](int I, int J) __attribute__((always_inline)) { return (live_bits >> (8 * I + J)) & 1ull; };

  // ---- 1a. blocks (I, J <= I) of C and G, dealt out round robin over the
  // waves, every block formed (the masks zero the dead ones, so later phases
  // read them without tests).  K_J Q_I^T comes back with column
  // i = 16 I + lr and rows j = 16 J + 4 lg + r: per lane exactly the
  // A-operand elements of C_IJ in C U (row i, K = nodes j), and likewise
  // K_J K_I^T gives the B-operand elements of G_IJ^T.
  const int nblk = tri(nt);
  // block k -> (I, J), J <= I, without a loop (k < 36)
  auto row_of = [](int k) __attribute__((always_inline)) {
    return (k >= 1) + (k >= 3) + (k >= 6) + (k >= 10) + (k >= 15) + (k >= 21) + (k >= 28);
  };
  // Two blocks side by side: every LDS read of both first (their operand
  // fragments, mask words and decays), then the four MFMA chains
  // interleaved, then masking.
  auto form2 = [&](int k0, int k1, f32x4 (&cv)[2], f32x4 (&gv)[2]) __attribute__((always_inline)) {
    int I[2], J[2];
    I[0] = row_of(k0);
    J[0] = k0 - tri(I[0]);
    I[1] = row_of(k1);
    J[1] = k1 - tri(I[1]);
    bf16x8 kj[2][KS], qi[2][KS], ki[2][KS];
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        kj[b][ks] = frag(s_k, kTile * J[b], ks);
        qi[b][ks] = frag(s_q, kTile * I[b], ks);
        ki[b][ks] = frag(s_k, kTile * I[b], ks);
      }
    // loads clamped into the arrays and the values selected, so that no
    // LDS read sits under a branch
    uint64_t mw0[2];
    float cl0[2], b00[2];
    f32x4 clj[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int i = kTile * I[b] + lr;
      mw0[b] = s_mask[min(i, tm - 1) * W + (J[b] >> 2)];
      cl0[b] = s_cl[i];
      b00[b] = s_beta[min(i, tm - 1)];
      clj[b] = *reinterpret_cast<const f32x4*>(s_cl + kTile * J[b] + 4 * lg);
    }
    f32x4 qk[2], kk[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) qk[b] = kk[b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        qk[b] = mfma16(kj[b][ks], qi[b][ks], qk[b]);
        kk[b] = mfma16(kj[b][ks], ki[b][ks], kk[b]);
      }
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const bool iv = kTile * I[b] + lr < T;
      const uint64_t mw = iv ? mw0[b] : 0ull;
      const unsigned mb = (unsigned)(mw >> ((J[b] & 3) * kTile + 4 * lg)) & 0xFu;
      const float cli = iv ? cl0[b] : 0.f, bi = iv ? b00[b] : 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bool m = (mb >> r) & 1u;
        const bool self = J[b] == I[b] && 4 * lg + r == lr;
        const float dec = __builtin_amdgcn_exp2f(cli - clj[b][r]);
        const float c = (dec * a.q_scale) * qk[b][r], g = (bi * dec) * kk[b][r];
        cv[b][r] = m ? c : 0.f;
        gv[b][r] = (m && !self) ? g : 0.f;
      }
    }
  };
  auto store = [&](int k, const f32x4& cv, const f32x4& gv) __attribute__((always_inline)) {
    const int I = row_of(k), J = k - tri(I);
    put_half(s_c, pair_row(I) + J / 2, J & 1, cv);
    if (J < I) {
      put_half(s_g, gpair_row(I) + J / 2, J & 1, -gv);   // stored negated: products accumulate -G
    } else {
      *reinterpret_cast<f32x4*>(s_gin + I * kTile * kTile + lr * kTile + 4 * lg) = gv;
      // the halves no block fills: (I, I + 1) of C for even I, (I, I) of G for odd I
      if ((I & 1) == 0) zero_half(s_c, pair_row(I) + I / 2, 1);
      else zero_half(s_g, gpair_row(I) + I / 2, 1);
    }
  };
  // ---- 1a'. the in-tile inverses (I + G_II)^{-1}, by the wave that formed
  // block (I, I) (block k = I (I + 3) / 2 goes to wave k % 8), from the
  // in-tile block it stored itself: forward substitution on the identity
  // over the tile's in-tile strict ancestors, in index order (lane s of each
  // 16-lane row holds x_s and broadcasts it by DPP row_newbcast).  Lane
  // (lr, lg) then holds row lr, columns 4 lg .. + 3 of the inverse: the A
  // operand of a 16x16x16 product.
  auto ainv_body = [&](auto Ic) __attribute__((always_inline)) {
    constexpr int I = decltype(Ic)::value;
    const float* gi = s_gin + I * kTile * kTile + lr * kTile;
    const f32x4 g0 = *reinterpret_cast<const f32x4*>(gi), g1 = *reinterpret_cast<const f32x4*>(gi + 4),
                g2 = *reinterpret_cast<const f32x4*>(gi + 8), g3 = *reinterpret_cast<const f32x4*>(gi + 12);
    const unsigned tin = __builtin_amdgcn_readfirstlane(s_tin[I]);
    f32x4 y;
#pragma unroll
    for (int r = 0; r < 4; ++r) y[r] = (4 * lg + r == lr) ? 1.f : 0.f;
    auto sub = [&](auto sc) __attribute__((always_inline)) {
      constexpr int s = decltype(sc)::value;
      if ((tin >> s) & 1u) {   // uniform
        const float gis = s < 4 ? g0[s & 3] : s < 8 ? g1[s & 3] : s < 12 ? g2[s & 3] : g3[s & 3];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float xs = __int_as_float(
              __builtin_amdgcn_mov_dpp(__float_as_int(y[r]), 0x150 + s, 0xF, 0xF, false));
          y[r] -= gis * xs;
        }
      }
    };
    static_for<kTile>(sub);
    bf16x4 hi, lo;
    split4_bf16(y, hi, lo);
    *reinterpret_cast<bf16x4*>(s_ainv + I * 1024 + lane * 8) = hi;
    *reinterpret_cast<bf16x4*>(s_ainv + I * 1024 + 512 + lane * 8) = lo;
  };
  auto make_ainv = [&](auto Ic) __attribute__((always_inline)) {
    constexpr int I = decltype(Ic)::value;
    constexpr int kdiag = I * (I + 3) / 2;
    if (I >= nt || kdiag % kDenseWaves != wave) return;   // uniform
    ainv_body(Ic);
  };
  // 1a of a full tree (node tiles 0..NTM - 1) for wave w, a compile-time
  // constant: blocks w, w + 8, ... and the inverses of the diagonal blocks
  // among them, with no branch, so that the compiler can overlap the reads
  // of one pair of blocks with the products of the one before
  // Blocks (I, J0 .. J0 + NJ - 1) of one row, I, J0, NJ compile-time
  // constants: the row's Q_I and K_I fragments are read once for all of them
  // (K_J once per block), then their MFMA chains run side by side.
  auto form_row = [&](auto Ic, auto J0c, auto NJc) __attribute__((always_inline)) {
    constexpr int I = decltype(Ic)::value, J0 = decltype(J0c)::value, NJ = decltype(NJc)::value;
    bf16x8 qi[KS], ki[KS], kj[NJ][KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      qi[ks] = frag(s_q, kTile * I, ks);
      ki[ks] = frag(s_k, kTile * I, ks);
#pragma unroll
      for (int b = 0; b < NJ; ++b) kj[b][ks] = frag(s_k, kTile * (J0 + b), ks);
    }
    const int i = kTile * I + lr;
    const bool iv = i < T;
    const float cli = iv ? s_cl[i] : 0.f, bi = iv ? s_beta[min(i, tm - 1)] : 0.f;
    uint64_t mw[W];
#pragma unroll
    for (int w = 0; w < W; ++w) mw[w] = iv ? s_mask[min(i, tm - 1) * W + w] : 0ull;
    f32x4 qk[NJ], kk[NJ];
#pragma unroll
    for (int b = 0; b < NJ; ++b) qk[b] = kk[b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int b = 0; b < NJ; ++b) {
        qk[b] = mfma16(kj[b][ks], qi[ks], qk[b]);
        kk[b] = mfma16(kj[b][ks], ki[ks], kk[b]);
      }
#pragma unroll
    for (int b = 0; b < NJ; ++b) {
      const int J = J0 + b;
      const f32x4 clj = *reinterpret_cast<const f32x4*>(s_cl + kTile * J + 4 * lg);
      const unsigned mb = (unsigned)(mw[J >> 2] >> ((J & 3) * kTile + 4 * lg)) & 0xFu;
      f32x4 cv, gv;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bool m = (mb >> r) & 1u;
        const bool self = J == I && 4 * lg + r == lr;
        const float dec = __builtin_amdgcn_exp2f(cli - clj[r]);
        const float c = (dec * a.q_scale) * qk[b][r], g = (bi * dec) * kk[b][r];
        cv[r] = m ? c : 0.f;
        gv[r] = (m && !self) ? g : 0.f;
      }
      store(tri(I) + J, cv, gv);
    }
  };
  // 1a of a full tree (node tiles 0..NTM - 1) for wave w, a compile-time
  // constant, with no branch.  The rows are paired (I, NTM - 1 - I): 9
  // blocks a pair, split over two waves so that each takes a contiguous run
  // of one row's blocks (sharing that row's fragments), plus at most a run
  // of the other row, and the diagonal blocks' inverses go with them:
  //   w0: (7, 0..3) (0, 0)      w1: (7, 4..7)
  //   w2: (6, 0..4)             w3: (6, 5..6) (1, 0..1)
  //   w4: (5, 0..3) (2, 0)      w5: (5, 4..5) (2, 1..2)
  //   w6: (4, 0..4)             w7: (3, 0..3)
  auto phase1a_full = [&](auto Wc) __attribute__((always_inline)) {
    constexpr int w = decltype(Wc)::value;
    static_assert(NTM == 8 && kDenseWaves == 8, "the row pairing is written for 8 tiles and 8 waves");
    using std::integral_constant;
    constexpr int p = w / 2, hi = NTM - 1 - p, lo = p;   // the row pair
    // the split of the pair's 9 blocks: (run of row hi) + (run of row lo)
    constexpr int hiJ0[8] = {0, 4, 0, 5, 0, 4, 0, 0};
    constexpr int hiN[8] = {4, 4, 5, 2, 4, 2, 5, 0};
    constexpr int loJ0[8] = {0, 0, 0, 0, 0, 1, 0, 0};
    constexpr int loN[8] = {1, 0, 0, 2, 1, 2, 0, 4};
    if constexpr (hiN[w] > 0) form_row(integral_constant<int, hi>{}, integral_constant<int, hiJ0[w]>{},
                                       integral_constant<int, hiN[w]>{});
    if constexpr (loN[w] > 0) form_row(integral_constant<int, lo>{}, integral_constant<int, loJ0[w]>{},
                                       integral_constant<int, loN[w]>{});
    // the inverses of the diagonal blocks this wave formed
    if constexpr (hiN[w] > 0 && hiJ0[w] + hiN[w] - 1 == hi) ainv_body(integral_constant<int, hi>{});
    if constexpr (loN[w] > 0 && loJ0[w] + loN[w] - 1 == lo) ainv_body(integral_constant<int, lo>{});
  };
  if (nt == NTM) {   // uniform
    switch (wave) {   // uniform
      case 0: phase1a_full(std::integral_constant<int, 0>{}); break;
      case 1: phase1a_full(std::integral_constant<int, 1>{}); break;
      case 2: phase1a_full(std::integral_constant<int, 2>{}); break;
      case 3: phase1a_full(std::integral_constant<int, 3>{}); break;
      case 4: phase1a_full(std::integral_constant<int, 4>{}); break;
      case 5: phase1a_full(std::integral_constant<int, 5>{}); break;
      case 6: phase1a_full(std::integral_constant<int, 6>{}); break;
      default: phase1a_full(std::integral_constant<int, 7>{}); break;
    }
  } else {
    // two blocks per step (block k goes to wave k % 8)
    for (int k = wave; k < nblk; k += 2 * kDenseWaves) {   // uniform
      const int k2 = k + kDenseWaves;
      f32x4 cv[2], gv[2];
      form2(k, min(k2, nblk - 1), cv, gv);
      store(k, cv[0], gv[0]);
      if (k2 < nblk) store(k2, cv[1], gv[1]);
    }
    static_for<NTM>(make_ainv);
  }
  TL_TRACE_POINT(a, 8);

  // ---- 1b. B0 = Q S^T and SK = K S^T for this wave's channels, all node tiles
  // (rows = nodes 16 I + 4 lg + r, column = channel 16 wave + lr)
  f32x4 b0[NTM];
  bf16x8 rph[NTM / 2], rpl[NTM / 2];   // R as B operands, tiles paired (K = nodes of 2 P, 2 P + 1)
#pragma unroll
  for (int P = 0; P < NTM / 2; ++P) {
    rph[P] = bf16x8{};
    rpl[P] = bf16x8{};
  }
  bf16x8 shi[KS], slo[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) split8_bf16(sraw[ks][0], sraw[ks][1], shi[ks], slo[ks]);

  TL_TRACE_POINT(a, 9);
  auto tile1b = [&](auto Ic) __attribute__((always_inline)) {
    constexpr int I = decltype(Ic)::value;
    f32x4 bb = f32x4{0.f, 0.f, 0.f, 0.f}, sk = bb;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const bf16x8 qf = frag(s_q, kTile * I, ks), kf = frag(s_k, kTile * I, ks);
      bb = mfma16(qf, shi[ks], bb);
      sk = mfma16(kf, shi[ks], sk);
      bb = mfma16(qf, slo[ks], bb);
      sk = mfma16(kf, slo[ks], sk);
    }
    b0[I] = bb;
    // R_j = beta_j (v_j - P_j (S k_j)); zero past the tree (those columns of
    // A meet only zero coefficients, and must stay finite)
    const f32x4 clj = *reinterpret_cast<const f32x4*>(s_cl + kTile * I + 4 * lg);
    const f32x4 bj = *reinterpret_cast<const f32x4*>(s_beta + kTile * I + 4 * lg);
    f32x4 rv;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const bool jv = kTile * I + 4 * lg + r < T;
      rv[r] = jv ? bj[r] * ((float)vv[I][r] - __builtin_amdgcn_exp2f(clj[r]) * sk[r]) : 0.f;
    }
    set_half(rph[I / 2], rpl[I / 2], I & 1, rv);
  };
  auto tile1b_any = [&](auto Ic) __attribute__((always_inline)) {
    if (decltype(Ic)::value < nt) tile1b(Ic);   // uniform
    else b0[decltype(Ic)::value] = f32x4{0.f, 0.f, 0.f, 0.f};
  };
  // (a branch-free form for full trees measured slower: 1b's tiles are
  // independent, and the compiler hoisted reads of later tiles at the cost
  // of registers)
  static_for<NTM>(tile1b_any);
  TL_TRACE_POINT(a, 10);
  lds_barrier();   // C, G and the in-tile inverses are in LDS; K and Q are dead
  TL_TRACE_POINT(a, 4);

  // ---- 2. column block J = wave of A = (I + G)^{-1}: for I = J, J + 1, ...
  //   Y_I = delta_IJ - sum_{J <= K < I} G_IK X_K,   X_I = (I + G_II)^{-1} Y_I.
  // Y and X come out of the products with row i (node of tile I) and column j
  // (node of tile J): per lane exactly the B-operand elements of a product
  // whose K index is i, so X_K feeds the later sums and Y feeds the in-tile
  // inverse without any transposition.  The sums run over pairs of node
  // tiles (16x16x32, the stored -G as A operands).  With X_I the wave also
  // forms block (I, J) of C A = sum_{J <= K <= I} C_IK X_K (the stored C as A
  // operands), which goes to LDS in A-operand layout for phase 3, over the
  // dead K and Q rows: O = C U = (C A) R.  Every block (I, J <= I) of C A is
  // written, zero where no ancestor relation (an entry (i, j) of C A needs
  // j in Anc(k) u {k} and k in Anc(i) u {i} for some k).
  // pair P of row I of C (tiles 2 P, 2 P + 1) holds a nonzero block
  auto pair_live = [&](int I, int P) __attribute__((always_inline)) {
    return live(I, 2 * P) || (2 * P + 1 <= I && live(I, 2 * P + 1));
  };
  // Column block J, generic form: any tree, dead blocks skipped.
  auto column_any = [&](int J) __attribute__((always_inline)) {
    bf16x8 xph[NTM / 2], xpl[NTM / 2];   // X_K as B operands, tiles paired (zero below J)
#pragma unroll
    for (int P = 0; P < NTM / 2; ++P) {
      xph[P] = bf16x8{};
      xpl[P] = bf16x8{};
    }
    auto step_tile = [&](auto Ic) __attribute__((always_inline)) {
      constexpr int I = decltype(Ic)::value;
      if (I < J || I >= nt) return;   // uniform
      const int pa = pair_row(I) + J / 2;
      if (I == J && (I & 1) == 0) zero_half(s_a, pa, 1);   // (I, I + 1): never a block
      if (!live(I, J)) {              // A_IJ = 0, (C A)_IJ = 0 (and X_I stays zero)
        zero_half(s_a, pa, J & 1);
        return;
      }
      const bf16x4 ah = *reinterpret_cast<const bf16x4*>(s_ainv + I * 1024 + lane * 8);
      const bf16x4 al = *reinterpret_cast<const bf16x4*>(s_ainv + I * 1024 + 512 + lane * 8);
      f32x4 y, y2 = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int r = 0; r < 4; ++r) y[r] = (I == J && 4 * lg + r == lr) ? 1.f : 0.f;
      // - sum_{K < I} G_IK X_K over tile pairs (X_K is zero below J and where
      // A_KJ is; the half K = I of the last pair is zero), G stored negated
#pragma unroll
      for (int P = 0; 2 * P < I; ++P) {
        if (2 * P + 1 < J) continue;   // uniform: both halves of X are zero
        bf16x8 gh, gl;
        get_pair(s_g, gpair_row(I) + P, gh, gl);
        y = mfma16(gh, xph[P], y);
        y2 = mfma16(gl, xph[P], y2);
        y = mfma16(gh, xpl[P], y);
      }
      y += y2;
      bf16x4 yh, yl;
      split4_bf16(y, yh, yl);
      f32x4 x = mfma16k(ah, yh, f32x4{0.f, 0.f, 0.f, 0.f});
      f32x4 x2 = mfma16k(al, yh, f32x4{0.f, 0.f, 0.f, 0.f});
      x = mfma16k(ah, yl, x);
      x += x2;
      set_half(xph[I / 2], xpl[I / 2], I & 1, x);
      // (C A)_IJ = sum_{J <= K <= I} C_IK X_K over tile pairs (the half
      // K = I + 1 of the last pair is zero in both), formed transposed: with
      // the X fragments as A operands and the stored C as B operands, the
      // product comes back with column i and rows j, so a lane holds row i
      // of (C A)_IJ at the K positions of its lane group, which is its part
      // of the A operand of phase 3 as it stands (no transposition)
      f32x4 ca = f32x4{0.f, 0.f, 0.f, 0.f}, ca2 = ca;
#pragma unroll
      for (int P = 0; 2 * P <= I; ++P) {
        if (2 * P + 1 < J || !pair_live(I, P)) continue;   // uniform: X or C is zero
        bf16x8 ch, cl;
        get_pair(s_c, pair_row(I) + P, ch, cl);
        ca = mfma16(xph[P], ch, ca);
        ca2 = mfma16(xpl[P], ch, ca2);
        ca = mfma16(xph[P], cl, ca);
      }
      put_half(s_a, pa, J & 1, ca + ca2);
    };
    static_for<NTM>(step_tile);
  };
  // Column block J of a full tree (node tiles 0..NTM - 1), J a compile-time
  // constant: no branch at all, so the compiler can issue a step's LDS reads
  // (G, the in-tile inverse, C) during the products of the step before.
  // Dead blocks are formed too: every term of their products pairs a zero
  // coefficient with a zero X entry or the other way round, so they come
  // out exactly zero for finite inputs (a non-finite input of the request
  // may spread through them, within the bounds the delta rule documents).
  auto column_full = [&](auto Jc) __attribute__((always_inline)) {
    constexpr int J = decltype(Jc)::value;
    bf16x8 xph[NTM / 2], xpl[NTM / 2];
#pragma unroll
    for (int P = 0; P < NTM / 2; ++P) {
      xph[P] = bf16x8{};
      xpl[P] = bf16x8{};
    }
    auto step_tile = [&](auto Ic) __attribute__((always_inline)) {
      constexpr int I = decltype(Ic)::value;
      if constexpr (I >= J) {
        constexpr int pa = pair_row(I) + J / 2;
        if constexpr (I == J && (I & 1) == 0) zero_half(s_a, pa, 1);   // (I, I + 1): never a block
        const bf16x4 ah = *reinterpret_cast<const bf16x4*>(s_ainv + I * 1024 + lane * 8);
        const bf16x4 al = *reinterpret_cast<const bf16x4*>(s_ainv + I * 1024 + 512 + lane * 8);
        f32x4 y, y2 = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int r = 0; r < 4; ++r) y[r] = (I == J && 4 * lg + r == lr) ? 1.f : 0.f;
#pragma unroll
        for (int P = (J & ~1) / 2; 2 * P < I; ++P) {   // pairs below J / 2 hold zero X
          bf16x8 gh, gl;
          get_pair(s_g, gpair_row(I) + P, gh, gl);
          y = mfma16(gh, xph[P], y);
          y2 = mfma16(gl, xph[P], y2);
          y = mfma16(gh, xpl[P], y);
        }
        y += y2;
        bf16x4 yh, yl;
        split4_bf16(y, yh, yl);
        f32x4 x = mfma16k(ah, yh, f32x4{0.f, 0.f, 0.f, 0.f});
        f32x4 x2 = mfma16k(al, yh, f32x4{0.f, 0.f, 0.f, 0.f});
        x = mfma16k(ah, yl, x);
        x += x2;
        set_half(xph[I / 2], xpl[I / 2], I & 1, x);
        f32x4 ca = f32x4{0.f, 0.f, 0.f, 0.f}, ca2 = ca;
#pragma unroll
        for (int P = (J & ~1) / 2; 2 * P <= I; ++P) {
          bf16x8 ch, cl;
          get_pair(s_c, pair_row(I) + P, ch, cl);
          ca = mfma16(xph[P], ch, ca);
          ca2 = mfma16(xpl[P], ch, ca2);
          ca = mfma16(xph[P], cl, ca);
        }
        put_half(s_a, pa, J & 1, ca + ca2);
      }
    };
    static_for<NTM>(step_tile);
  };
  if (nt == NTM) {   // uniform
    switch (wave) {   // uniform
      case 0: column_full(std::integral_constant<int, 0>{}); break;
      case 1: column_full(std::integral_constant<int, 1>{}); break;
      case 2: column_full(std::integral_constant<int, 2>{}); break;
      case 3: column_full(std::integral_constant<int, 3>{}); break;
      case 4: column_full(std::integral_constant<int, 4>{}); break;
      case 5: column_full(std::integral_constant<int, 5>{}); break;
      case 6: column_full(std::integral_constant<int, 6>{}); break;
      default: column_full(std::integral_constant<int, 7>{}); break;
    }
    static_assert(NTM == kDenseWaves, "one column block per wave");
  } else if (wave < nt) {   // uniform
    column_any(wave);
  }
  lds_barrier();   // C A is in LDS
  TL_TRACE_POINT(a, 5);

  // ---- 3. O = q_scale P B0 + (C A) R for this wave's channels: 16x16x32
  // products over pairs of node tiles, C A read whole from LDS, R the
  // register fragments
  float* obase = a.out + (size_t)(off + 4 * lg) * v_row + (size_t)h * D + kTile * wave + lr;
  // tile I of phase 3; ALL: every row of the tile is a node (no store test)
  // and dead pairs are read as the zeros they hold (no branch)
  auto tile3 = [&](auto Ic, auto ALLc) __attribute__((always_inline)) {
    constexpr int I = decltype(Ic)::value;
    constexpr bool ALL = decltype(ALLc)::value;
    f32x4 o = f32x4{0.f, 0.f, 0.f, 0.f}, o2 = o;
#pragma unroll
    for (int P = 0; 2 * P <= I; ++P) {
      if (!ALL && !pair_live(I, P)) continue;   // uniform
      bf16x8 ah, al;
      get_pair(s_a, pair_row(I) + P, ah, al);
      o = mfma16(ah, rph[P], o);
      o2 = mfma16(ah, rpl[P], o2);
      o = mfma16(al, rph[P], o);
    }
    const f32x4 cli = *reinterpret_cast<const f32x4*>(s_cl + kTile * I + 4 * lg);
    float* orow = obase + (size_t)(kTile * I) * v_row;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float v = a.q_scale * __builtin_amdgcn_exp2f(cli[r]) * b0[I][r] + (o[r] + o2[r]);
      if (ALL || kTile * I + 4 * lg + r < T) __builtin_nontemporal_store(v, orow + (size_t)r * v_row);
    }
  };
  auto tile3_all = [&](auto Ic) __attribute__((always_inline)) { tile3(Ic, std::true_type{}); };
  auto tile3_any = [&](auto Ic) __attribute__((always_inline)) {
    if (decltype(Ic)::value < nt) tile3(Ic, std::false_type{});   // uniform
  };
  if (T == kTile * NTM) static_for<NTM>(tile3_all);   // uniform
  else static_for<NTM>(tile3_any);
  TL_TRACE_POINT(a, 15);
#ifdef TL_TRACE
  if (a.trace && threadIdx.x == 0) a.trace[(size_t)blockIdx.x * 16 + 14] = (long long)__builtin_readcyclecounter();
#endif
}

int verify_gdn_dense_lds_bytes(int tm) { return dense_layout(tm, tm > 64 ? 2 : 1).total; }

template <int W>
static tl_status launch_dense_w(const VerifyArgs& a, hipStream_t stream) {
  const int lds = dense_layout(a.tm, W).total;
  if (lds > 160 * 1024) return TL_EUNSUPPORTED;
  const long blocks = 8 * (((long)a.batch * a.Hk + 7) / 8) * (a.Hv / a.Hk);
  if (blocks == 0) return TL_OK;
  if (blocks > 0x7fffffffL) return TL_EINVAL;
  auto kern = verify_gdn_dense_kernel<W>;
  if (lds > 64 * 1024) {
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                            hipFuncAttributeMaxDynamicSharedMemorySize, lds) != hipSuccess)
      return TL_EHIP;
  }
  VerifyArgs b = a;
  b.lds_bytes = lds;
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kDenseThreads), lds, stream, b);
  return hipGetLastError() == hipSuccess ? TL_OK : TL_EHIP;
}

tl_status launch_verify_gdn_dense(const tl_problem& p, const VerifyArgs& a, hipStream_t stream) {
  if (p.mode != TL_MODE_GDN || p.in_dtype != TL_BF16 || p.d_k != 128 || a.tm > 128)
    return TL_EUNSUPPORTED;
  return a.tm > 64 ? launch_dense_w<2>(a, stream) : launch_dense_w<1>(a, stream);
}

}  // namespace tl
