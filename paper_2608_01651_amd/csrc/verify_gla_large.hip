// Verify, gated linear attention on MFMA over trees of 65..256 nodes.
//
// One workgroup per (request, v-head), one wave per 16-row value tile of the
// stored state (8 waves at d = 128; at d < 128 spare waves only help form
// coefficients).  Theorem 1 with U = V (§4.1):
//   O^T = q_scale P .* (S Q^T) + V^T C^T,
//   C_ij = [j in Anc(i) u {i}] 2^(cl_i - cl_j) (q_i . k_j) q_scale,
// with cl the cumulative log2-decay along the root path.  Nodes are taken in
// tiles of 16 in index order, which is topological, so the ancestors of tile
// I lie in tiles 0..I.
//
// Everything the node tiles read is made resident on chip before the first
// tile, so the tile walk issues no global load: its only global accesses are
// the output stores.  (Loads and stores share one completion counter on this
// GPU, and the compiler waits for every outstanding access wherever a loaded
// register is first read while a store is pending; a walk that read
// prefetched rows waited for the previous tile's stores at every tile.)
//
//  prologue  batch 1: wave 0 loads the parents and gates and forms the
//            topology alone (M+ rows, cl, per-tile OR of the M+ rows; pointer
//            jumping in LDS with no workgroup barrier) while the other
//            waves copy, by direct global -> LDS copies, the V rows (into the
//            K region; rows past T repeat row T - 1) and the Q rows; every
//            value wave loads its state rows (registers).  Each value wave
//            then reads its V^T operand fragments of every 32-node chunk out
//            of the staged rows with LDS transpose reads (ds_read_b64_tr_b16;
//            32 VGPRs at 256 nodes), entries of nodes >= T set to zero.
//            Batch 2 copies the K rows over the staged V rows.
//  tile I    (a) coefficients: the ancestor columns of a tile are cut into
//            chunks of 32 nodes (tiles 2c, 2c + 1) and dealt out to the waves
//            by half chunk (one 16-node tile J).  A half chunk is one K_J
//            Q_I^T MFMA chain; its output lanes hold B-operand elements of
//            V^T C^T, so it is masked, decayed, split into bf16 hi + lo and
//            stored in operand order.  Half chunks without an ancestor of the
//            tile (tile masks) are stored as zeros without MFMA work.
//            (b) per value wave: S Q_I^T with the state split into bf16
//            hi + lo (two MFMA chains), plus V^T C^T over the chunks that hold
//            an ancestor (two chains, hi and lo), scaled, added and stored.
//  When LDS holds two chunk buffers, (a) of tile I + 1 and (b) of tile I share
//  one step and one barrier; otherwise (node caps of 240 and 256 at d = 128)
//  they alternate between two barriers.
#include <hip/hip_runtime.h>

#include "tl_device.h"
#include "tl_kernels.h"
#include "verify_common.h"

namespace tl {

__host__ __device__ constexpr int gla_large_waves(int D) { return D / kTile > kWaves ? D / kTile : kWaves; }

// Rows of the K region: the K rows of tm nodes, and before them the V rows of
// every 32-node chunk a tree of tm nodes reads.
__host__ __device__ constexpr int gla_large_rows(int tm) { return (tm + 31) & ~31; }

struct GlaLargeLayout {
  int flag, cl, mask, tmask, kst, qst, frag, fragsz, frag2, total;
};

// Where the chunk operands of odd node tiles go.  kBufTwo: a second buffer
// after the first; kBufK: the start of the K region.
// A wave reads the K rows of tile J once, into registers, when it forms the
// half chunks of tile J (the diagonal block is never empty), so when the
// chunks of tile I are formed the K rows of tiles 0..I - 1 are dead, and
// the I + 1 KB the operands of an odd tile I take lie below the rows of tile
// I at d >= 64.
enum GlaLargeBuf { kBufTwo = 1, kBufK = 2 };

// LDS layout (bytes); identical on host and device.
__host__ __device__ inline GlaLargeLayout gla_large_layout(int D, int tm, int W, int buf) {
  GlaLargeLayout L;
  int o = 0;
  L.flag = o;  o += 16;                                  // the tree is malformed
  L.cl = o;    o += align16(tm * 4);                     // cumulative log2-decay (0 past T)
  L.mask = o;  o += tm * W * 8;                          // M+ rows (0 past T)
  L.tmask = o; o += align16((tm / kTile) * W * 8);       // OR of the M+ rows per node tile
  L.kst = o;   o += gla_large_rows(tm) * D * 2;          // K rows | staged V rows, swizzled bf16
  L.qst = o;   o += tm * D * 2;                          // Q rows, swizzled bf16
  L.frag = o;                                            // chunk operands | topology scratch
  L.fragsz = ((tm + 31) / 32) * 2 * 1024;                // chunks of tiles 0..I: C hi, C lo
  const int topo = 64 * W * (4 + 4) + 64 * W * W * 8;   // wave_topology_jump scratch
  const int fr = (buf == kBufTwo ? 2 : 1) * L.fragsz;
  o += align16(fr > topo ? fr : topo);
  L.frag2 = buf == kBufTwo ? L.frag + L.fragsz : (buf == kBufK ? L.kst : L.frag);
  L.total = o;
  return L;
}

// The buffering of a problem: two buffers where LDS holds them, else the K
// region (d >= 64; at d = 32 two buffers always fit).
__host__ __device__ inline int gla_large_buf(int D, int tm, int W) {
  return gla_large_layout(D, tm, W, kBufTwo).total <= 160 * 1024 ? kBufTwo : kBufK;
}

template <int D, int W, int BUF>
__global__ __launch_bounds__(64 * gla_large_waves(D)) __attribute__((amdgpu_waves_per_eu(2, 2))) void verify_gla_large_kernel(VerifyArgs a) {
  constexpr int NW = gla_large_waves(D);
  constexpr int NT = 64 * NW;
  constexpr int VT = D / kTile;            // value tiles: wave w < VT owns rows 16w..16w+15
  constexpr int KS = D / 32;
  constexpr int CPRK = D / 8;              // 16-byte chunks per row
  constexpr int NCH = 2 * W;               // 32-node chunks of the largest tree
  constexpr float kLog2e = 1.4426950408889634f;
  constexpr int NE = W;                    // nodes per lane of wave 0 (node cap <= 64 W)
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
  const GlaLargeLayout L = gla_large_layout(D, tm, W, BUF);
  float* s_cl = reinterpret_cast<float*>(tl_lds + L.cl);
  uint64_t* s_mask = reinterpret_cast<uint64_t*>(tl_lds + L.mask);
  uint64_t* s_tmask = reinterpret_cast<uint64_t*>(tl_lds + L.tmask);
  __bf16* s_k = reinterpret_cast<__bf16*>(tl_lds + L.kst);
  __bf16* s_q = reinterpret_cast<__bf16*>(tl_lds + L.qst);
  unsigned char* s_frag = tl_lds + L.frag;

  const size_t qk_row = (size_t)a.Hk * D, v_row = (size_t)a.Hv * D;
  const __bf16* Qb = reinterpret_cast<const __bf16*>(a.q) + (size_t)off * qk_row + (size_t)hq * D;
  const __bf16* Kb = reinterpret_cast<const __bf16*>(a.k) + (size_t)off * qk_row + (size_t)hq * D;
  const __bf16* Vb = reinterpret_cast<const __bf16*>(a.v) + (size_t)off * v_row + (size_t)h * D;

  // ---- prologue, batch 1: wave 0 loads the parents and gates and its
  // state rows, and forms the topology alone (wave_topology_jump, no
  // workgroup barrier) while waves 1.. copy the V and Q rows into LDS and
  // load their state rows.  Copy position p = base + lane holds 16-byte
  // chunk swz(r, p % CPRK) of row r = p / CPRK.  The copies are inline
  // assembly, which the compiler does not count, so wave 0, whose waits the
  // compiler places, issues none.
  TL_TRACE_POINT(a, 1);
  // The parents, gates and copies are issued at raised wave priority and the
  // state rows at the normal one, so that every wave's copies reach the
  // memory queue before any wave's state rows (the older waves would
  // otherwise win the issue arbitration with their state loads).
  __builtin_amdgcn_s_setprio(2);
  int par[NE];
  float gx[NE];
  if (wave == 0) {   // uniform
#pragma unroll
    for (int e = 0; e < NE; ++e) {   // unconditional loads, clamped to the tree
      const int i = off + min(lane + 64 * e, T - 1);
      par[e] = a.parent[i];
      gx[e] = a.g[(size_t)i * a.Hv + h];
    }
  }
  // the parents and gates enter this CU's memory queue ahead of the bulk
  // copies (a barrier without a memory wait: wave 0's loads are issued, not
  // complete)
  __builtin_amdgcn_s_barrier();
  const int TP = (T + 31) & ~31;   // V rows of every chunk the tree reads
  if (wave > 0) {   // uniform
    for (int base = (wave - 1) * 64; base < TP * CPRK; base += NT - 64) {   // TP * CPRK is a multiple of 64
      const int p = base + lane, r = p / CPRK, c = swz<CPRK>(r, p % CPRK);
      copy16_to_lds_async(Vb + (size_t)min(r, T - 1) * v_row + c * 8, s_k + (size_t)base * 8);
    }
    for (int base = (wave - 1) * 64; base < T * CPRK; base += NT - 64) {
      const int p = base + lane;
      if (p < T * CPRK) {
        const int r = p / CPRK, c = swz<CPRK>(r, p % CPRK);
        copy16_to_lds_async(Qb + (size_t)r * qk_row + c * 8, s_q + (size_t)base * 8);
      }
    }
  }
  // the wave's state rows last: the batch's wait leaves them in flight, and
  // they are first read after the topology
  f32x4 sraw[KS][2];
  auto load_state = [&]() __attribute__((always_inline)) {
    const float* row = a.state + ((size_t)sidx * a.Hv + h) * D * D + (size_t)(kTile * wave + lr) * D;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      sraw[ks][0] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(row + ks * 32 + 8 * lg));
      sraw[ks][1] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(row + ks * 32 + 8 * lg + 4));
    }
  };
  // unconditional where every wave is a value wave, so that the compiler's
  // count of outstanding loads is the same on every path and its waits for
  // the parents and gates do not take in the state rows
  __builtin_amdgcn_s_setprio(0);   // the state rows at the normal priority
  if constexpr (VT == NW) load_state();
  else if (vw) load_state();
  // ---- topology by wave 0: M+ rows, cl, per-tile OR of the M+ rows (rows
  // past T: zero masks and decays)
  int* s_flag = reinterpret_cast<int*>(tl_lds + L.flag);
  if (wave == 0) {   // uniform
    // the parents and gates have landed; the state rows issued after them
    // stay in flight through the topology
    if constexpr (VT == NW) wait_vmem_below<2 * KS>();
    for (int x = lane; x < (tm / kTile) * W; x += 64) s_tmask[x] = 0;
    int* s_jmp = reinterpret_cast<int*>(s_frag);
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
        if (i < tm) {
          s_cl[i] = i < T ? cl[e] * kLog2e : 0.f;
#pragma unroll
          for (int w = 0; w < W; ++w) s_mask[i * W + w] = i < T ? msk[e][w] : 0ull;
          if (i < T) {
            const int I = i / kTile;
#pragma unroll
            for (int w = 0; w < W; ++w)
              if (msk[e][w]) atomicOr(reinterpret_cast<unsigned long long*>(&s_tmask[I * W + w]),
                                      (unsigned long long)msk[e][w]);
          }
        }
      }
    }
  }
  TL_TRACE_POINT(a, 13);
  // batch 1 but the state rows has landed (loads complete in issue order; a
  // wait the compiler sees)
  if constexpr (VT == NW) wait_vmem_below<2 * KS>();
  else if (vw) wait_vmem_below<2 * KS>();
  else wait_vmem_below<0>();
  lds_barrier();          // staged V rows, Q rows and the topology are visible
  TL_TRACE_POINT(a, 2);
  if (*s_flag) {   // uniform: a malformed tree (reported by wave 0)
    wait_vmem();   // the state rows land before the block retires
    return;
  }

  // the wave's V^T operand fragments of every chunk: lane (lg, lr) names row
  // 4 lg + lr / 4 of a 16-node half chunk and columns 16 w + 4 (lr % 4) .. + 3,
  // so it receives value channel 16 w + lr of nodes 4 lg .. 4 lg + 3 of that
  // half (K positions kpos(lg, 0..3) and kpos(lg, 4..7) for the two halves)
  bf16x8 vreg[NCH];
  {
    const int nch = TP / 32;   // chunks that hold a node (uniform)
    const int vrow_l = 4 * lg + (lr >> 2);
    const int col = kTile * (vw ? wave : 0) + 4 * (lr & 3);
    const int vo = vrow_l * D * 2 + swz<CPRK>(vrow_l, col >> 3) * 16 + (col & 7) * 2;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      bf16x8 f = bf16x8{};
      if (vw && c < nch) {   // uniform
        // rows 32 c + vrow_l and 32 c + 16 + vrow_l keep the swizzle key of
        // row vrow_l (32 c and 16 are multiples of CPRK)
        const bf16x4 x0 = lds_read_tr16(s_k, vo + (32 * c) * D * 2);
        const bf16x4 x1 = lds_read_tr16(s_k, vo + (32 * c + 16) * D * 2);
        f = bf16x8{x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
        // nodes >= T carry copies of row T - 1; their coefficients are zero,
        // and zero values keep a non-finite input of node T - 1 from reaching
        // other nodes through them
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int n = 32 * c + (e < 4 ? 4 * lg + e : 16 + 4 * lg + (e - 4));
          if (n >= T) f[e] = (__bf16)0.f;
        }
      }
      vreg[c] = f;
    }
  }
  TL_TRACE_POINT(a, 11);
  lds_barrier();   // every wave has read the staged V rows

  // ---- batch 2: K rows over the staged V rows
  for (int base = wave * 64; base < T * CPRK; base += NT) {   // uniform
    const int p = base + lane;
    if (p < T * CPRK) {
      const int r = p / CPRK, c = swz<CPRK>(r, p % CPRK);
      copy16_to_lds_async(Kb + (size_t)r * qk_row + c * 8, s_k + (size_t)base * 8);
    }
  }
  TL_TRACE_POINT(a, 3);
  // the wave's state rows, split into bf16 hi + lo MFMA A operands
  bf16x8 shi[KS], slo[KS];
  if (vw) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) split8_bf16(sraw[ks][0], sraw[ks][1], shi[ks], slo[ks]);
  }
  TL_TRACE_POINT(a, 14);
  wait_vmem();     // batch 2 (the K rows) has landed
  lds_barrier();   // K rows are visible; the topology scratch is dead
  TL_TRACE_POINT(a, 4);

  // operand fragment of row R + lr (R a multiple of 16), K chunk ks, of a
  // swizzled LDS matrix
  const int key = lr & (CPRK - 1);
  const int fo_row = lr * D * 2;
  auto frag = [&](const __bf16* base, int R, int ks) __attribute__((always_inline)) {
    const unsigned char* p = reinterpret_cast<const unsigned char*>(base) + R * D * 2 + fo_row;
    return *reinterpret_cast<const bf16x8*>(p + (((4 * ks + lg) ^ key) * 16));
  };
  // the tile masks, word x in lane x (at most 64 words), and 32 bits of tile
  // I's mask starting at node 32 c, read across lanes (uniform)
  const uint64_t tmv = lane < (tm / kTile) * W ? s_tmask[lane] : 0ull;
  auto tile_bits32 = [&](int I, int c) __attribute__((always_inline)) {
    const int x = I * W + (c >> 1);
    return (c & 1) ? (unsigned)__builtin_amdgcn_readlane((int)(uint32_t)(tmv >> 32), x)
                   : (unsigned)__builtin_amdgcn_readlane((int)(uint32_t)tmv, x);
  };

  // (a) coefficient chunks of tile I into buf: half chunk J (tiles 0 ..
  // 2 (I / 2) + 1) goes to wave J % NW, so a wave always forms the same half
  // chunks and keeps their K_J fragments in registers once read (kreg slot
  // J / NW).  Half chunks without an ancestor of the tile are stored as
  // zeros, so the value work reads every chunk 0 .. I / 2 without a test.
  // Operand layout [chunk][hi | lo][lane] 16 bytes, half J & 1 in bytes
  // 8 (J & 1) .. + 7.  qf holds the Q fragments of tile I.  The tile index is
  // a compile-time constant (the tile loop is unrolled), so every chunk
  // count is one too.
  constexpr int NJ = 4 * W;                     // node tiles of the largest tree
  constexpr int NKS = (NJ + NW - 1) / NW;       // half chunks per wave
  bf16x8 kreg[NKS][KS];
  auto chunks = [&](auto Ic, const bf16x8 (&qf)[KS], unsigned char* buf) __attribute__((always_inline)) {
    constexpr int I = decltype(Ic)::value;
    constexpr int nh = 2 * (I / 2 + 1);
    const int i = kTile * I + lr;
    const float cli = s_cl[i];
#pragma unroll
    for (int sl = 0; sl < NKS; ++sl) {
      const int J = wave + sl * NW;
      if (J >= nh) break;   // uniform
      const int c = J >> 1, hf = J & 1;
      const unsigned bits = (tile_bits32(I, c) >> (hf * kTile)) & 0xFFFFu;
      float cv[4] = {0.f, 0.f, 0.f, 0.f};
      if (J <= I && bits) {   // uniform
        if (J == I) {         // first use of tile J (its own diagonal block is never empty)
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) kreg[sl][ks] = frag(s_k, kTile * J, ks);
        }
        f32x4 qk = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) qk = mfma16(kreg[sl][ks], qf[ks], qk);   // rows j, column i
        const uint64_t mw = s_mask[i * W + (J >> 2)];   // M+ row of node i (zero past T)
        const f32x4 clj = *reinterpret_cast<const f32x4*>(s_cl + kTile * J + 4 * lg);
        const unsigned mb = (unsigned)(mw >> ((J & 3) * kTile + 4 * lg)) & 0xFu;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          cv[r] = ((mb >> r) & 1u) ? (__builtin_amdgcn_exp2f(cli - clj[r]) * a.q_scale) * qk[r] : 0.f;
      }
      uint32_t cw[4];   // hi01 hi23, lo01 lo23
      split2_bf16(cv[0], cv[1], cw[0], cw[2]);
      split2_bf16(cv[2], cv[3], cw[1], cw[3]);
      unsigned char* pc = buf + ((c * 2) * 64 + lane) * 16 + hf * 8;
      *reinterpret_cast<uint2*>(pc) = uint2{cw[0], cw[1]};
      *reinterpret_cast<uint2*>(pc + 1024) = uint2{cw[2], cw[3]};
    }
  };
  // Q fragments of tile I (B operand, columns = the tile's nodes)
  auto load_qf = [&](int I, bf16x8 (&qf)[KS]) __attribute__((always_inline)) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = frag(s_q, kTile * I, ks);
  };

  // (b) value rows of this wave for tile I, from the chunk operands in buf:
  // the operands of chunks 0 .. I / 2 are all requested first, so their LDS
  // latency overlaps one another and the state term's products
  float* obase = a.out + (size_t)off * v_row + (size_t)h * D + kTile * wave + 4 * lg;
  auto value_work = [&](auto Ic, const bf16x8 (&qf)[KS], const unsigned char* buf) __attribute__((always_inline)) {
    constexpr int I = decltype(Ic)::value;
    constexpr int NC = I / 2 + 1;
    const int i = kTile * I + lr;
    bf16x8 ch[NC], cl[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const unsigned char* pc = buf + ((c * 2) * 64 + lane) * 16;
      ch[c] = *reinterpret_cast<const bf16x8*>(pc);
      cl[c] = *reinterpret_cast<const bf16x8*>(pc + 1024);
    }
    const float cli = s_cl[i];
    f32x4 b0h = f32x4{0.f, 0.f, 0.f, 0.f}, b0l = b0h, acc = b0h, acc2 = b0h;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      b0h = mfma16(shi[ks], qf[ks], b0h);
      b0l = mfma16(slo[ks], qf[ks], b0l);
    }
#pragma unroll
    for (int c = 0; c < NC; ++c) {   // V^T from registers
      acc = mfma16(vreg[c], ch[c], acc);
      acc2 = mfma16(vreg[c], cl[c], acc2);
    }
    if (i < T) {
      const float ps = __builtin_amdgcn_exp2f(cli) * a.q_scale;
      f32x4 o;
#pragma unroll
      for (int r = 0; r < 4; ++r) o[r] = ps * (b0h[r] + b0l[r]) + (acc[r] + acc2[r]);
      store_out<false>(obase + (size_t)i * v_row, o);
    }
  };

  // Each step forms the chunks of tile I + 1 (buffer (I + 1) & 1, free since
  // the previous barrier) while the value work of tile I reads buffer I & 1:
  // one barrier per tile.  Every wave reads the Q fragments of the tile whose
  // chunks it forms and keeps them for that tile's value work.
  const int nt = (T + kTile - 1) / kTile;
  bf16x8 qcur[KS], qnext[KS];
  load_qf(0, qcur);
  chunks(std::integral_constant<int, 0>{}, qcur, s_frag);
  lds_barrier();
  TL_TRACE_POINT(a, 5);
  auto step = [&](auto Ic) __attribute__((always_inline)) {
    constexpr int I = decltype(Ic)::value;
    if (I >= nt) return;   // uniform
    unsigned char* bnext = ((I + 1) & 1) ? tl_lds + L.frag2 : s_frag;
    const unsigned char* bcur = (I & 1) ? tl_lds + L.frag2 : s_frag;
    if (I == 9) TL_TRACE_POINT(a, 7);
    if constexpr (I + 1 < NJ) {
      if (I + 1 < nt) {
        load_qf(I + 1, qnext);
        chunks(std::integral_constant<int, I + 1>{}, qnext, bnext);
      }
    }
    if (I == 9) TL_TRACE_POINT(a, 8);
    if (vw) value_work(Ic, qcur, bcur);
    if (I == 9) TL_TRACE_POINT(a, 9);
    lds_barrier();   // chunks of tile I + 1 visible; buffer I & 1 free again
    if (I == 9) TL_TRACE_POINT(a, 10);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qcur[ks] = qnext[ks];
    if (I == 0) TL_TRACE_POINT(a, 6);
  };
  static_for<NJ>(step);
  TL_TRACE_POINT(a, 15);
}

// LDS bytes of the kernel for a node cap.
int verify_gla_large_lds_bytes(int d, int tm) {
  const int W = tm > 128 ? 4 : (tm > 64 ? 2 : 1);
  return gla_large_layout(d, tm, W, gla_large_buf(d, tm, W)).total;
}

template <int D, int W, int BUF>
static tl_status launch_gla_large_one(const VerifyArgs& a, hipStream_t stream) {
  const int lds = gla_large_layout(D, a.tm, W, BUF).total;
  if (lds > 160 * 1024) return TL_EUNSUPPORTED;
  const long blocks = 8 * (((long)a.batch * a.Hk + 7) / 8) * (a.Hv / a.Hk);
  if (blocks == 0) return TL_OK;
  if (blocks > 0x7fffffffL) return TL_EINVAL;
  auto kern = verify_gla_large_kernel<D, W, BUF>;
  if (lds > 64 * 1024) {
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                            hipFuncAttributeMaxDynamicSharedMemorySize, lds) != hipSuccess)
      return TL_EHIP;
  }
  VerifyArgs b = a;
  b.lds_bytes = lds;
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(64 * gla_large_waves(D)), lds, stream, b);
  return hipGetLastError() == hipSuccess ? TL_OK : TL_EHIP;
}

template <int D, int W>
static tl_status launch_gla_large_buf(const VerifyArgs& a, hipStream_t stream) {
  if (gla_large_buf(D, a.tm, W) == kBufTwo) return launch_gla_large_one<D, W, kBufTwo>(a, stream);
  if constexpr (D >= 64) return launch_gla_large_one<D, W, kBufK>(a, stream);
  return TL_EUNSUPPORTED;
}

template <int D>
static tl_status launch_gla_large_w(const VerifyArgs& a, hipStream_t stream) {
  if (a.tm > 128) return launch_gla_large_buf<D, 4>(a, stream);
  return launch_gla_large_buf<D, 2>(a, stream);
}

tl_status launch_verify_gla_large(const tl_problem& p, const VerifyArgs& a, hipStream_t stream) {
  if (a.tm <= 64 || a.tm > 256) return TL_EUNSUPPORTED;
  switch (p.d_k) {
    case 32: return launch_gla_large_w<32>(a, stream);
    case 64: return launch_gla_large_w<64>(a, stream);
    case 128: return launch_gla_large_w<128>(a, stream);
    default: return TL_EUNSUPPORTED;
  }
}

}  // namespace tl
