// Device helpers shared by the verify, commit and topology kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>

#include <stdint.h>
#include <type_traits>
#include <utility>

#include "treelin.h"

// Phase time stamps for trace builds (-DTL_TRACE): thread 0 of each block
// records the 100 MHz wall clock at point k (and, at point 0, its compute unit
// id in slot 12).  Empty in normal builds.
#ifdef TL_TRACE
#define TL_TRACE_POINT(args, k)                                                           \
  do {                                                                                    \
    if ((args).trace && threadIdx.x == 0) {                                               \
      (args).trace[(size_t)blockIdx.x * 16 + (k)] = wall_clock64();                       \
      if ((k) == 0) (args).trace[(size_t)blockIdx.x * 16 + 12] = __smid();                \
    }                                                                                     \
  } while (0)
#else
#define TL_TRACE_POINT(args, k) \
  do {                          \
  } while (0)
#endif

namespace tl {

// f(std::integral_constant<int, J>{}) for J = 0 .. N-1, in order.  Always
// inlined: the bodies are whole kernel phases, and an outlined call would
// give them a stack frame and the calling convention's register budget.
template <class F, int... J>
__device__ __attribute__((always_inline)) inline void static_for_seq(F& f, std::integer_sequence<int, J...>) {
  (f(std::integral_constant<int, J>{}), ...);
}
template <int N, class F>
__device__ __attribute__((always_inline)) inline void static_for(F& f) {
  static_for_seq(f, std::make_integer_sequence<int, N>{});
}

constexpr int kThreads = 256;      // every kernel runs 4 wave64s per workgroup
constexpr int kWaves = kThreads / 64;
constexpr int kMaxNodes = 256;     // one node per thread in the topology pass
constexpr int kTile = 16;          // nodes per MFMA tile (M or N of 16x16x32)

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// error reporting: first failing request wins (compare-and-swap from 0)
// ---------------------------------------------------------------------------
__device__ inline void report(int32_t* dev_err, int32_t code) {
  if (dev_err) atomicCAS(dev_err, 0, code);
}

// ---------------------------------------------------------------------------
// number formats
// ---------------------------------------------------------------------------
__device__ inline float bf2f(__bf16 x) { return (float)x; }

// fp32 -> bf16 hi + bf16 lo with hi + lo == x to about 2^-17 relative
// (the two-term bf16 split: hi is x rounded to nearest even, lo is the
// rounded residual).
__device__ inline void split_bf16(float x, __bf16& hi, __bf16& lo) {
  hi = (__bf16)x;
  lo = (__bf16)(x - (float)hi);
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Two fp32 values -> bf16 hi pair + bf16 lo pair (one 32-bit word each,
// element 0 in the low half).  hi is x with its low 16 bits cleared
// (truncation), so x - hi is exact in fp32 and |x - hi| < 2^-7 |x|; lo is that
// remainder rounded to nearest, so hi + lo == x to 2^-16 relative.  Costs one
// byte permute for the two hi values, and an AND, a subtract and half a
// convert per value for lo.
__device__ inline void split2_bf16(float x0, float x1, uint32_t& hi, uint32_t& lo) {
  const uint32_t b0 = __float_as_uint(x0), b1 = __float_as_uint(x1);
  hi = __builtin_amdgcn_perm(b1, b0, 0x07060302u);   // high halves of b0 (low) and b1 (high)
  const float l0 = x0 - __uint_as_float(b0 & 0xffff0000u);
  const float l1 = x1 - __uint_as_float(b1 & 0xffff0000u);
  lo = __builtin_bit_cast(uint32_t, bf16x2{(__bf16)l0, (__bf16)l1});
}

// Eight fp32 values (a then b) -> bf16x8 hi and lo operands (split2_bf16).
__device__ inline void split8_bf16(const f32x4& a, const f32x4& b, bf16x8& hi, bf16x8& lo) {
  uint32_t h0, h1, h2, h3, l0, l1, l2, l3;
  split2_bf16(a[0], a[1], h0, l0);
  split2_bf16(a[2], a[3], h1, l1);
  split2_bf16(b[0], b[1], h2, l2);
  split2_bf16(b[2], b[3], h3, l3);
  hi = __builtin_bit_cast(bf16x8, u32x4{h0, h1, h2, h3});
  lo = __builtin_bit_cast(bf16x8, u32x4{l0, l1, l2, l3});
}

// 4 consecutive inputs as floats, from bf16 or fp32 storage.
template <bool F32IN>
__device__ inline f32x4 load4(const void* base, size_t idx) {
  if constexpr (F32IN) {
    return *reinterpret_cast<const f32x4*>(reinterpret_cast<const float*>(base) + idx);
  } else {
    bf16x4 t = *reinterpret_cast<const bf16x4*>(reinterpret_cast<const __bf16*>(base) + idx);
    return f32x4{(float)t[0], (float)t[1], (float)t[2], (float)t[3]};
  }
}

template <bool F32IN>
__device__ inline float load1(const void* base, size_t idx) {
  if constexpr (F32IN) return reinterpret_cast<const float*>(base)[idx];
  else return (float)reinterpret_cast<const __bf16*>(base)[idx];
}

// ---------------------------------------------------------------------------
// MFMA 16x16x32 bf16 (gfx950).  D = A (16 x 32) * B (32 x 16) + C.
// Lane l supplies A row (l % 16) and B column (l % 16), each as 8 values of
// the K range owned by lane group l / 16; D comes back as rows
// 4*(l/16) .. 4*(l/16)+3 of column (l % 16).
//
// The K index is only a contraction index, so any assignment of the 32 K
// positions to (lane group, element) works as long as A and B use the same
// one.  Every operand here uses kpos(): group gq holds columns 4gq..4gq+3 and
// 16+4gq..16+4gq+3 of the 32-wide K chunk, so one 16-byte row load of four
// lane groups covers 64 contiguous bytes of fp32 state.
// ---------------------------------------------------------------------------
__device__ inline int kpos(int gq, int e) { return (e < 4) ? (4 * gq + e) : (16 + 4 * gq + (e - 4)); }

__device__ inline f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Operand fragment (8 bf16) of row `row` (already offset to the row start)
// for K chunk `ks`, lane group gq: two 8-byte loads.  Returns zeros if !ok.
__device__ inline bf16x8 frag_bf16(const __bf16* row, int ks, int gq, bool ok) {
  bf16x8 r;
  if (ok) {
    bf16x4 a = *reinterpret_cast<const bf16x4*>(row + ks * 32 + 4 * gq);
    bf16x4 b = *reinterpret_cast<const bf16x4*>(row + ks * 32 + 16 + 4 * gq);
    r = bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  } else {
    __bf16 z = (__bf16)0.0f;
    r = bf16x8{z, z, z, z, z, z, z, z};
  }
  return r;
}

// ---------------------------------------------------------------------------
// request bounds and forest checks (uniform per workgroup)
// ---------------------------------------------------------------------------
struct Request {
  int off;   // first global row
  int T;     // node count
};

// Returns false (and reports TL_EBADTREE) for decreasing offsets or
// T_b > max_nodes.  Uniform across the block.
__device__ inline bool load_request(const int32_t* node_offsets, int b, int max_nodes,
                                    int32_t* dev_err, Request& r) {
  int o0 = node_offsets[b], o1 = node_offsets[b + 1];
  r.off = o0;
  r.T = o1 - o0;
  if (o0 < 0 || r.T < 0 || r.T > max_nodes) {
    if (threadIdx.x == 0) report(dev_err, TL_EBADTREE);
    return false;
  }
  return true;
}

// ---------------------------------------------------------------------------
// Topology over the parent array (one thread per node).
//
// `par` is node i's parent (any value for threads i >= T).
// Computes, for node i = threadIdx.x < T:
//   depth  = number of strict ancestors,
//   cl     = sum of x over Anc(i) u {i}   (the cumulative log-decay when x = g,
//            so P_i = exp(cl_i) and P_i / P_j = exp(cl_i - cl_j)),
//   mask   = the M+ row of i as W little-endian 64-bit words.
// Every node first walks up its own root path through the parents in LDS,
// folding in one ancestor per step with no barrier (a wave runs as many steps
// as its deepest node needs), for at most kTopoWalk steps.  A node's state
// then covers the path segment from itself up to (excluding) jmp.  Nodes
// still short of the root finish by pointer jumping over those segments:
// after round r a node has folded in 2^r segments above it, and all threads
// take part in every barrier.  Returns false (uniformly) if any parent
// breaks the parent-before-child order.  Scratch arrays need kThreads
// entries (kThreads * W words for the mask scratch).
// ---------------------------------------------------------------------------
constexpr int kTopoWalk = 16;

template <int W, bool WANT_MASK>
__device__ inline bool build_topology(int par, int T, float x,
                                      int32_t* s_jmp, float* s_acc, int32_t* s_cnt,
                                      uint64_t* s_msk, int& depth, float& cl,
                                      uint64_t (&mask)[W]) {
  const int i = threadIdx.x;
  const bool live = i < T;
  const bool bad = live && !(par == -1 || (par >= 0 && par < i));
  if (live) {   // parents and own values, read by the walks of descendants
    s_jmp[i] = par;
    s_acc[i] = x;
  }
  if (__syncthreads_or(bad)) return false;   // also orders the stores above before the walks

  int jmp = live ? par : -1;
  int cnt = 1;
  cl = x;
#pragma unroll
  for (int w = 0; w < W; ++w) mask[w] = (live && WANT_MASK && (i >> 6) == w) ? (1ull << (i & 63)) : 0ull;

  for (int s = 0; s < kTopoWalk; ++s) {
    if (__ballot(jmp >= 0) == 0ull) break;   // uniform: every node of the wave is at its root
    if (jmp >= 0) {
      const int up = s_jmp[jmp];
      cl += s_acc[jmp];
      cnt += 1;
      if constexpr (WANT_MASK) {
#pragma unroll
        for (int w = 0; w < W; ++w) mask[w] |= ((jmp >> 6) == w) ? (1ull << (jmp & 63)) : 0ull;
      }
      jmp = up;
    }
  }

  // the loop test is a barrier: no segment is stored before every walk (and
  // every partner read of the previous round) is done
  while (__syncthreads_or(live && jmp >= 0)) {
    if (live) {
      s_jmp[i] = jmp;
      s_acc[i] = cl;
      s_cnt[i] = cnt;
      if constexpr (WANT_MASK) {
#pragma unroll
        for (int w = 0; w < W; ++w) s_msk[w * kThreads + i] = mask[w];
      }
    }
    __syncthreads();
    if (live && jmp >= 0) {
      cl += s_acc[jmp];
      cnt += s_cnt[jmp];
      if constexpr (WANT_MASK) {
#pragma unroll
        for (int w = 0; w < W; ++w) mask[w] |= s_msk[w * kThreads + jmp];
      }
      jmp = s_jmp[jmp];
    }
  }
  depth = cnt - 1;
  return true;
}

// The same topology (cl and the M+ rows of build_topology) formed by one wave
// alone, with no workgroup barrier, so that it can run while the other waves
// of the workgroup are held up issuing their copies: lane l holds nodes
// l + 64 e (e < NE), so T <= 64 NE.  Pointer jumping: a node's state (cl,
// mask) covers the path segment from itself up to (excluding) jmp; each
// round every node publishes its state, then folds in the state published
// at jmp, doubling its segment, so a tree of depth d takes ceil(log2(d + 1))
// rounds.  The LDS accesses of one wave take effect in program order, so no
// round needs a barrier (with one wave, rounds are cheaper than the
// one-ancestor-per-step walks build_topology starts with).  Ancestors have
// smaller indices, so the M+ row of node n has no bit in words above n / 64:
// those words are not published, and a fold takes a word from jmp only if
// jmp published it.  Scratch: s_jmp and s_acc of 64 NE entries, s_msk of
// W * 64 NE words (word-major, so that a publish writes consecutive words).
// Returns false (uniformly over the wave) if a parent breaks the
// parent-before-child order.
template <int W, int NE>
__device__ inline bool wave_topology_jump(const int (&par)[NE], const float (&x)[NE], int T,
                                          int32_t* s_jmp, float* s_acc, uint64_t* s_msk,
                                          float (&cl)[NE], uint64_t (&mask)[NE][W]) {
  static_assert(NE <= W, "node l + 64 e has its bit in word e");
  const int lane = threadIdx.x & 63;
  bool bad = false;
  int jmp[NE];
#pragma unroll
  for (int e = 0; e < NE; ++e) {
    const int i = lane + 64 * e;
    const bool live = i < T;
    bad |= live && !(par[e] == -1 || (par[e] >= 0 && par[e] < i));
    jmp[e] = live ? par[e] : -1;
    cl[e] = x[e];
#pragma unroll
    for (int w = 0; w < W; ++w) mask[e][w] = (live && e == w) ? (1ull << lane) : 0ull;
  }
  if (__ballot(bad)) return false;   // before any read through a parent

  auto pending = [&]() __attribute__((always_inline)) {
    bool any = false;
#pragma unroll
    for (int e = 0; e < NE; ++e) any |= jmp[e] >= 0;
    return __ballot(any) != 0ull;
  };
  while (pending()) {
#pragma unroll
    for (int e = 0; e < NE; ++e) {   // publish
      const int i = lane + 64 * e;
      if (i < T) {
        s_jmp[i] = jmp[e];
        s_acc[i] = cl[e];
#pragma unroll
        for (int w = 0; w <= e; ++w) s_msk[w * 64 * NE + i] = mask[e][w];
      }
    }
#pragma unroll
    for (int e = 0; e < NE; ++e) {   // fold in the segment above
      if (jmp[e] >= 0) {
        const int j = jmp[e];
        cl[e] += s_acc[j];
#pragma unroll
        for (int w = 0; w <= e; ++w) {
          const uint64_t m = s_msk[w * 64 * NE + j];   // in bounds; stale where w > j / 64
          if (w <= (j >> 6)) mask[e][w] |= m;
        }
        jmp[e] = s_jmp[j];
      }
    }
  }
  return true;
}

}  // namespace tl

namespace tl {

// Number of set bits of the W-word mask m strictly below bit j.
template <int W>
__device__ inline int popc_below(const uint64_t (&m)[W], int j) {
  int c = 0;
#pragma unroll
  for (int w = 0; w < W; ++w) {
    if (64 * w + 64 <= j) c += __popcll(m[w]);
    else if (64 * w <= j) c += __popcll(m[w] & ((1ull << (j - 64 * w)) - 1ull));
  }
  return c;
}

// ---------------------------------------------------------------------------
// Direct global -> LDS copies (gfx950 global_load_lds_dwordx4): each lane's
// 16 bytes land at lds_base + 16 * lane, without passing through registers.
// `lds_base` must be the same for the whole wave.
// ---------------------------------------------------------------------------
__device__ inline void copy16_to_lds(const void* gsrc, void* lds_base) {
  __builtin_amdgcn_global_load_lds(gsrc, (__attribute__((address_space(3))) void*)lds_base, 16, 0, 0);
}

// The same copy, issued as inline assembly: the compiler does not see the
// LDS write, so it does not hold later LDS accesses behind every outstanding
// load of the wave (it would have to assume they alias the copy).  The
// caller must wait for completion itself (wait_vmem / wait_vmem_below)
// before the copied bytes are read.  M0 (the LDS base of the copy) is saved
// and restored around it, so no register the compiler owns is changed; one
// wait state separates each M0 write from the next instruction that reads it.
// NT selects the non-temporal (streaming) cache policy, for data read once.
template <bool NT = false>
__device__ inline void copy16_to_lds_async(const void* gsrc, void* lds_base) {
  const uint32_t m0v = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)lds_base);
  uint32_t saved;
  if constexpr (NT)
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, off nt\n\t"
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0"
        : "=&s"(saved)
        : "v"(gsrc), "s"(m0v)
        : "memory");
  else
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, off\n\t"
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0"
        : "=&s"(saved)
        : "v"(gsrc), "s"(m0v)
        : "memory");
}

// Sum of x over aligned groups of N lanes (N = 2, 4, 8, 16 or 32); every lane
// of a group receives the same total.  Within a row of 16 lanes the partners
// come from DPP (quad xor 1, quad xor 2, half-row mirror, row mirror: each
// step adds two partial sums that cover disjoint lanes); the two rows of a
// 32-lane group are joined by one swizzle (lane xor 16).  Every lane of the
// wave must be active.
template <int N>
__device__ inline float group_sum(float x) {
  static_assert(N == 2 || N == 4 || N == 8 || N == 16 || N == 32, "groups of 2, 4, 8, 16 or 32 lanes");
  auto dpp = [](float v, auto ctrl) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), decltype(ctrl)::value, 0xF, 0xF, true));
  };
  x += dpp(x, std::integral_constant<int, 0xB1>{});   // quad_perm [1, 0, 3, 2]
  if constexpr (N >= 4) x += dpp(x, std::integral_constant<int, 0x4E>{});   // quad_perm [2, 3, 0, 1]
  if constexpr (N >= 8) x += dpp(x, std::integral_constant<int, 0x141>{});   // row_half_mirror
  if constexpr (N >= 16) x += dpp(x, std::integral_constant<int, 0x140>{});  // row_mirror
  if constexpr (N >= 32)   // bitmask swizzle: and 0x1f, or 0, xor 0x10
    x += __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(x), 0x401F));
  return x;
}

// The same for 4 bytes per lane (global_load_lds_dword): each active lane's
// dword lands at lds_base + 4 * lane; inactive lanes copy nothing.
__device__ inline void copy4_to_lds_async(const void* gsrc, void* lds_base) {
  const uint32_t m0v = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)lds_base);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dword %1, off\n\t"
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0"
      : "=&s"(saved)
      : "v"(gsrc), "s"(m0v)
      : "memory");
}

// Waits for every outstanding vector memory operation of this wave
// (including the direct-to-LDS copies).
__device__ inline void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Waits until at most N vector memory operations of this wave are
// outstanding.  Loads complete in issue order, so everything issued before
// the last N has landed (gfx9 encoding: vmcnt in bits 3:0 and 15:14, expcnt
// and lgkmcnt left at their maxima).
template <int N>
__device__ inline void wait_vmem_below() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// LDS transpose read of 16-bit data (gfx950 ds_read_b64_tr_b16).  Within
// each group of 16 lanes, lane s names 8 bytes (4 consecutive elements) at
// `byte_off`; lane s receives element (s % 4) of the chunks named by lanes
// s/4, s/4 + 4, s/4 + 8 and s/4 + 12 of its group, in that order.  So if
// lane s names row r0 + s/4, columns c0 + 4 (s % 4) .. + 3 of a row-major
// matrix, lane s gets column c0 + s of rows r0 .. r0 + 3: four consecutive
// K values of an MFMA operand row, read from K-major storage.
typedef short s16x4 __attribute__((ext_vector_type(4)));
__device__ inline bf16x4 lds_read_tr16(const void* lds_base, uint32_t byte_off) {
  typedef __attribute__((address_space(3))) s16x4* lp;
  const uint32_t a = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)lds_base + byte_off;
  return __builtin_bit_cast(bf16x4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lp)(uintptr_t)a));
}

// Output rows are written once and never read back by the kernel; NT
// selects the non-temporal (streaming) cache policy for them.
template <bool NT>
__device__ inline void store_out(float* p, const f32x4& v) {
  if constexpr (NT) __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(p));
  else *reinterpret_cast<f32x4*>(p) = v;
}

// Workgroup barrier for LDS data: this wave's LDS accesses complete, then
// s_barrier.  Unlike __syncthreads() it does not wait for the wave's
// outstanding global loads, so loads issued for later phases stay in flight.
__device__ inline void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Compiler-only fence: keeps the compiler from moving memory operations
// across this point (issue order matters for wait_vmem_below).
__device__ inline void issue_fence() { asm volatile("" ::: "memory"); }

// Rows of CPR 16-byte chunks are stored with chunk c at position
// c ^ (row & (CPR-1)) so that the same column of 16 consecutive rows falls in
// different LDS banks.
template <int CPR>
__device__ inline int swz(int row, int chunk) { return chunk ^ (row & (CPR - 1)); }

// Stage rows [0, T) of a strided bf16 matrix (row r at src + r * stride,
// CPR chunks of 8 values each) into swizzled LDS.  All threads of the block
// take part; completion needs wait_vmem() and a barrier.
template <int CPR>
__device__ inline void stage_rows_bf16(const __bf16* src, size_t stride, int T, __bf16* lds) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int total = T * CPR;
  for (int base = wave * 64; base < total; base += kThreads) {
    const int p = base + lane;
    if (p < total) {
      const int r = p / CPR, c = swz<CPR>(r, p % CPR);
      copy16_to_lds(src + (size_t)r * stride + c * 8, lds + (size_t)base * 8);
    }
  }
}

// 4 bf16 (8 bytes) at logical column `col` (multiple of 4) of row `row` of a
// swizzled LDS matrix.
template <int CPR>
__device__ inline bf16x4 lds_bf16x4(const __bf16* lds, int row, int col) {
  const int c = swz<CPR>(row, col >> 3);
  return *reinterpret_cast<const bf16x4*>(lds + ((size_t)row * CPR + c) * 8 + (col & 7));
}

// MFMA operand fragment (kpos() layout) of row `row`, K chunk ks, lane group
// gq, from a swizzled LDS matrix; zeros if !ok.
template <int CPR>
__device__ inline bf16x8 lds_frag(const __bf16* lds, int row, int ks, int gq, bool ok) {
  const bf16x4 x0 = lds_bf16x4<CPR>(lds, row, ks * 32 + 4 * gq);
  const bf16x4 x1 = lds_bf16x4<CPR>(lds, row, ks * 32 + 16 + 4 * gq);
  return ok ? bf16x8{x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]} : bf16x8{};
}

}  // namespace tl

namespace tl {

// 64-bit lane shuffle (two 32-bit ds_bpermute).
__device__ inline uint64_t shfl64(uint64_t x, int src) {
  const unsigned lo = __shfl((unsigned)(x & 0xffffffffull), src, 64);
  const unsigned hi = __shfl((unsigned)(x >> 32), src, 64);
  return ((uint64_t)hi << 32) | lo;
}

// Topology of a tree of T <= 64 nodes inside one wavefront, lane = node,
// by pointer jumping over lane shuffles (no LDS, no barriers).  `par` is the
// lane's parent (ignored for lanes >= T).  Returns false (for the whole
// wave) if a parent breaks the parent-before-child order; otherwise gives
// the lane's depth, its sum of x along the root path (inclusive) and its M+
// row as one 64-bit word.
__device__ inline bool wave_topology(int par, int T, float x, int& depth, float& cl,
                                     uint64_t& mask) {
  const int i = threadIdx.x & 63;
  const bool live = i < T;
  const bool bad = live && !(par == -1 || (par >= 0 && par < i));
  if (__ballot(bad)) return false;
  int jmp = live ? par : -1;
  int cnt = 1;
  cl = x;
  mask = live ? (1ull << i) : 0ull;
  while (__ballot(jmp >= 0)) {
    const int src = jmp >= 0 ? jmp : i;
    const uint64_t m2 = shfl64(mask, src);
    const float c2 = __shfl(cl, src, 64);
    const int n2 = __shfl(cnt, src, 64);
    const int j2 = __shfl(jmp, src, 64);
    if (jmp >= 0) {
      mask |= m2;
      cl += c2;
      cnt += n2;
      jmp = j2;
    }
  }
  depth = cnt - 1;
  return true;
}

}  // namespace tl
