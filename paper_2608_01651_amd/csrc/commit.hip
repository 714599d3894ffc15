// Accepted-path commit (§4.4, Eq. accepted-commit), one layer or many.
//
// S_new = P_a S_pre + (D_a K_a)^T U_a is, by Lemma 1, the post-update state
// of the terminal node a, i.e. the recurrence replayed along the accepted
// path from S_pre.  The kernel replays it in fp32, in place:
//   gated linear attention:  S <- gamma S + v k^T
//   gated delta rule:        u = beta (v - gamma S k),  S <- gamma S + u k^T
// (stored orientation: S is the slot's [d_v, d_k] matrix).  Rows of the
// stored state evolve independently under both rules (the delta rule's
// S k is a per-row dot product), so each block of rows is replayed on its
// own, and nothing crosses workgroups.  A workgroup checks the forest and the
// path before it writes anything, and every block is read before it is
// written; an empty path leaves the slot untouched.  The state is read and
// written once, with non-temporal loads and stores.
//
// The accepted path is shared by every recurrent layer, so §5.2 folds the
// commits of all layers into one launch; commit_layers_kernel does that, one
// workgroup per (layer, request, v-head).  There the path arrives as the
// sampled terminal node of each request (the path descriptor of §5.2) and is
// rebuilt on chip by walking the parents from it; accepted_path_kernel
// exports the same lists.
#include <hip/hip_runtime.h>

#include "tl_device.h"
#include "tl_kernels.h"

namespace tl {

constexpr int kCommitChunk = 32;   // path steps staged in LDS at a time

// A row of the stored state sits in LPR adjacent lanes, VPL values each, as
// CH chunks of 4: chunk c of lane l holds columns 4 (l % LPR) + 4 LPR c, so
// each load or store instruction covers whole 4 LPR-column runs of a row.
// The delta rule sums every row once per path step; at d >= 64 its rows are
// held by 8 lanes (three DPP steps per sum) instead of d / 4.
template <int D, int MODE>
struct CommitShape {
  static constexpr int ROWS = (D >= 64) ? 32 : D;   // state rows per streamed block
  static constexpr int NRB = D / ROWS;              // blocks per (request, v-head) slot
  static constexpr int VPL = (MODE == TL_MODE_GDN && D >= 64) ? D / 8 : 4;   // values per lane
  static constexpr int LPR = D / VPL;               // lanes per row
  static constexpr int CH = VPL / 4;                // 4-float chunks per lane and row
  static constexpr int RPP = kThreads / LPR;        // rows per pass of the workgroup
  static constexpr int PASSES = (ROWS + RPP - 1) / RPP;
};

// Block-wide OR through LDS: each wave's ballot goes to s_red[wave] (one
// array per use).  The barrier waits for LDS traffic only, so the state
// loads in flight stay in flight.
__device__ inline bool block_or_lds(bool pred, int* s_red) {
  const bool any = __ballot(pred) != 0ull;
  if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6] = any ? 1 : 0;
  lds_barrier();
  int r = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) r |= s_red[w];
  return r != 0;
}

// Accepted path ending at `term` (0 <= term < T) of a checked forest whose
// parents are in s_par: every thread walks the same root path (broadcast
// LDS reads; parents precede children, so the walk ends within T steps), and
// thread s keeps the node s steps above the terminal, which is path entry
// L - 1 - s.  Writes s_path[0 .. L) root first and returns L (uniform).
__device__ inline int path_to_root(int term, const int* s_par, int* s_path) {
  const int tid = threadIdx.x;
  int j = term, s = 0, mine = -1;
  while (j >= 0) {
    if (s == tid) mine = j;
    j = s_par[j];
    ++s;
  }
  if (tid < s) s_path[s - 1 - tid] = mine;
  lds_barrier();
  return s;
}

// Commit of one (request b, v-head h) slot of one layer.  TERMINAL: the path
// is the one ending at terminal[b] (-1: nothing accepted); otherwise it is
// path[path_offsets[b] .. path_offsets[b+1]-1], checked link by link.
//
// Order of the memory traffic: the parents (and the listed path) are
// requested first, then the state blocks, all unconditionally (a request
// that commits nothing points its state loads at one line), so the checks
// wait only for the former; the checks synchronise through LDS alone; the
// gates and k/v rows of the path then go out in one round trip, and the
// replay waits for everything.
//
// SPLIT workgroups share a slot: part `part` replays row blocks
// [part * NB, part * NB + NB), NB = NRB / SPLIT (each checks the forest and
// the path itself).
template <int MODE, int D, bool F32IN, bool TERMINAL, int SPLIT>
__device__ __attribute__((always_inline)) inline void commit_unit(
    const CommitCommon& a, const CommitLayer& ly, const int32_t* path_offsets,
    const int32_t* path, const int32_t* terminal, int b, int h, int part) {
  using SH = CommitShape<D, MODE>;
  constexpr int ROWS = SH::ROWS, NRB = SH::NRB, LPR = SH::LPR, CH = SH::CH, RPP = SH::RPP,
                PASSES = SH::PASSES;
  static_assert(NRB % SPLIT == 0, "a slot splits into whole row blocks");
  constexpr int NB = NRB / SPLIT;   // row blocks of this workgroup
  const int rb0 = part * NB;
  constexpr bool GDN = (MODE == TL_MODE_GDN);
  __shared__ __align__(16) float s_k[kCommitChunk * D];
  __shared__ __align__(16) float s_v[kCommitChunk * D];
  __shared__ float s_gam[kCommitChunk];
  __shared__ float s_beta[kCommitChunk];
  __shared__ int s_par[kMaxNodes];
  __shared__ int s_path[kMaxNodes];
  __shared__ int s_red[2 * kWaves];

  const int tid = threadIdx.x;
  TL_TRACE_POINT(a, 0);
  const int hq = h / (a.Hv / a.Hk);

  // the request's path descriptor and slot are requested together with its
  // node range (independent loads: one round trip, not three)
  int p0 = 0, Lp = 0, term = -1;
  if constexpr (TERMINAL) {
    term = terminal[b];
  } else {
    p0 = path_offsets[b];
    Lp = path_offsets[b + 1] - p0;
  }
  const int sidx = a.slot ? a.slot[b] : b;
  Request rq;
  if (!load_request(a.node_offsets, b, a.max_nodes, a.dev_err, rq)) return;
  const int T = rq.T, off = rq.off;
  if constexpr (!TERMINAL) {
    if (p0 < 0 || Lp < 0) {
      if (tid == 0) report(a.dev_err, TL_EINVAL);
      return;
    }
  }
  if (sidx < 0 || sidx >= a.num_slots) {
    if (tid == 0) report(a.dev_err, TL_EINVAL);
    return;
  }
  if (T == 0) {   // an empty request accepts nothing
    if ((TERMINAL ? term != -1 : Lp != 0) && tid == 0) report(a.dev_err, TL_EBADPATH);
    return;
  }
  TL_TRACE_POINT(a, 1);

  // parents and listed path nodes (clamped to valid rows; lanes past the end
  // are ignored)
  const int par = a.parent[off + min(tid, T - 1)];
  bool path_ok = true;
  int node = -1;
  if constexpr (!TERMINAL) {
    path_ok = !(Lp > T || (Lp > 0 && path == nullptr));
    const int32_t* np = (path_ok && Lp > 0) ? path + p0 + min(tid, Lp - 1) : a.parent + off;
    node = *np;
  }

  // state blocks; `keep` zeroes the offsets of a slot that is not written
  // (an AND with a value the compiler cannot see through, so the loads stay
  // one straight-line sequence)
  const bool need = TERMINAL ? term >= 0 : Lp > 0;
  float* Sp = ly.state + ((size_t)sidx * a.Hv + h) * D * D;
  const int col = (tid % LPR) * 4;   // column of the lane's chunk 0; chunk c is 4 LPR c further
  const int rsub = tid / LPR;
  uint32_t keep = need ? 0xffffffffu : 0u;
  asm volatile("" : "+v"(keep));
  using Block = f32x4[PASSES][CH];
  auto load_block = [&](int rb, Block& st) {
#pragma unroll
    for (int p = 0; p < PASSES; ++p) {
      const int row = min(p * RPP + rsub, ROWS - 1);
#pragma unroll
      for (int c = 0; c < CH; ++c) {
        const uint32_t o = (uint32_t)(((rb0 + rb) * ROWS + row) * D + col + 4 * LPR * c) & keep;
        st[p][c] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(Sp + o));
      }
    }
  };
  auto store_block = [&](int rb, const Block& st) {
#pragma unroll
    for (int p = 0; p < PASSES; ++p) {
      const int row = p * RPP + rsub;
      if (row < ROWS) {
#pragma unroll
        for (int c = 0; c < CH; ++c)
          __builtin_nontemporal_store(
              st[p][c], reinterpret_cast<f32x4*>(Sp + (size_t)((rb0 + rb) * ROWS + row) * D + col + 4 * LPR * c));
      }
    }
  };
  // gated linear attention keeps every block of the slot in registers (all
  // loads in flight at once); the delta rule needs more registers for its
  // row reductions and streams the blocks through two buffers
  constexpr int NBUF = GDN ? (NB < 2 ? NB : 2) : NB;
  Block sb[NBUF];
#pragma unroll
  for (int rb = 0; rb < NBUF; ++rb) load_block(rb, sb[rb]);

  // checks, through LDS only
  if (tid < T) s_par[tid] = par;
  if (!TERMINAL && tid < Lp && tid < kMaxNodes) s_path[tid] = node;
  const bool bad_tree = tid < T && !(par == -1 || (par >= 0 && par < tid));
  TL_TRACE_POINT(a, 2);
  if (block_or_lds(bad_tree, s_red)) {
    if (tid == 0) report(a.dev_err, TL_EBADTREE);
    return;
  }
  if constexpr (TERMINAL) {
    if (term < -1 || term >= T) {
      if (tid == 0) report(a.dev_err, TL_EBADPATH);
      return;
    }
    if (term < 0) return;
    Lp = path_to_root(term, s_par, s_path);
  } else {
    bool bad = !path_ok;
    if (!bad && tid < Lp) {
      const bool node_in = node >= 0 && node < T;
      bad = !node_in || s_par[node] != (tid == 0 ? -1 : s_path[tid - 1]);
    }
    if (block_or_lds(bad, s_red + kWaves)) {
      if (tid == 0) report(a.dev_err, TL_EBADPATH);
      return;
    }
    if (Lp == 0) return;
  }
  TL_TRACE_POINT(a, 3);

  const size_t qk_row = (size_t)a.Hk * D, v_row = (size_t)a.Hv * D;
  // stage path steps [c0, c0 + n): gates, k and v rows, in one round trip
  auto stage = [&](int c0, int n) {
    if (tid < n) {
      const size_t r = (size_t)(off + s_path[c0 + tid]);
      s_gam[tid] = __expf(ly.g[r * a.Hv + h]);
      if constexpr (GDN) s_beta[tid] = ly.beta[r * a.Hv + h];
    }
    for (int x = tid * 4; x < n * D; x += kThreads * 4) {
      const int t = x / D, e = x % D;
      const size_t r = (size_t)(off + s_path[c0 + t]);
      *reinterpret_cast<f32x4*>(s_k + x) = load4<F32IN>(ly.k, r * qk_row + (size_t)hq * D + e);
      *reinterpret_cast<f32x4*>(s_v + x) = load4<F32IN>(ly.v, r * v_row + (size_t)h * D + e);
    }
    __syncthreads();
  };
  // replay staged steps [0, n) on the rows of blocks rb .. rb + NR - 1, held
  // in sb[i0 .. i0 + NR); the blocks share each step's k row
  auto replay = [&](auto nr, int rb, int i0, int n) {
    constexpr int NR = decltype(nr)::value;
    if constexpr (!GDN) {
      static_assert(CH == 1, "one chunk per lane and row");
      for (int t = 0; t < n; ++t) {
        const float gam = s_gam[t];
        const f32x4 kv = *reinterpret_cast<const f32x4*>(s_k + t * D + col);
#pragma unroll
        for (int i = 0; i < NR; ++i) {
#pragma unroll
          for (int p = 0; p < PASSES; ++p) {
            const int row = p * RPP + rsub;
            const float vv = s_v[t * D + (rb0 + rb + i) * ROWS + (row < ROWS ? row : 0)];
            sb[i0 + i][p][0] = gam * sb[i0 + i][p][0] + vv * kv;
          }
        }
      }
    } else {
      // The rows are held as S / scale, scale = the product of the decays
      // so far, so that a step is one FMA per entry:
      //   S~ += (u / scale) k^T,  u = beta (v - scale (S~ k)).
      // When scale leaves [2^-32, 2^32] (or is not finite) it is folded into
      // the rows and restarts at 1; the final scale is folded in before the
      // rows are stored.  (Gated linear attention keeps gamma S + v k^T:
      // there the folding measured slower, its replay having no sums.)
      auto fold = [&](float f) {
#pragma unroll
        for (int i = 0; i < NR; ++i)
#pragma unroll
          for (int p = 0; p < PASSES; ++p)
#pragma unroll
            for (int c = 0; c < CH; ++c) sb[i0 + i][p][c] *= f;
      };
      float scale = 1.f;
      for (int t = 0; t < n; ++t) {
        scale *= s_gam[t];
        if (!(scale >= 0x1p-32f && scale <= 0x1p32f)) {   // uniform
          fold(scale);
          scale = 1.f;
        }
        const float inv = __builtin_amdgcn_rcpf(scale);
        const float bt = s_beta[t];
        f32x4 kv[CH];
#pragma unroll
        for (int c = 0; c < CH; ++c) kv[c] = *reinterpret_cast<const f32x4*>(s_k + t * D + col + 4 * LPR * c);
#pragma unroll
        for (int i = 0; i < NR; ++i) {
#pragma unroll
          for (int p = 0; p < PASSES; ++p) {
            f32x4* st = sb[i0 + i][p];
            f32x4 acc = st[0] * kv[0];
#pragma unroll
            for (int c = 1; c < CH; ++c) acc += st[c] * kv[c];
            float dot = (acc[0] + acc[1]) + (acc[2] + acc[3]);
            dot = group_sum<LPR>(dot);   // the row's LPR lanes
            const int row = p * RPP + rsub;
            const float vv = s_v[t * D + (rb0 + rb + i) * ROWS + (row < ROWS ? row : 0)];
            const float cf = bt * (vv - scale * dot) * inv;
#pragma unroll
            for (int c = 0; c < CH; ++c) st[c] += cf * kv[c];
          }
        }
      }
      fold(scale);
    }
  };
  using One = std::integral_constant<int, 1>;
  using All = std::integral_constant<int, NB>;

  // with the whole slot in registers, the path rows are requested only once
  // the slot has arrived: scattered row reads issued into the middle of the
  // launch-wide state stream slowed it down
  if constexpr (NBUF == NB) wait_vmem();
  if constexpr (GDN && NBUF == NB) {
    // every block is held: each chunk of steps is staged once and replayed
    // on all of them
    for (int c0 = 0; c0 < Lp; c0 += kCommitChunk) {
      const int n = min(kCommitChunk, Lp - c0);
      if (c0) __syncthreads();   // the previous chunk is fully consumed
      stage(c0, n);
      TL_TRACE_POINT(a, 4);
      replay(All{}, 0, 0, n);
    }
#pragma unroll
    for (int rb = 0; rb < NB; ++rb) store_block(rb, sb[rb]);
  } else if (Lp <= kCommitChunk) {
    stage(0, Lp);
#pragma unroll
    for (int rb = 0; rb < NB; ++rb) {
      replay(One{}, rb, rb % NBUF, Lp);
      store_block(rb, sb[rb % NBUF]);
      if (rb + NBUF < NB) load_block(rb + NBUF, sb[rb % NBUF]);
    }
  } else {
    // long paths through streamed blocks: the steps are staged chunk by
    // chunk for every block
#pragma unroll
    for (int rb = 0; rb < NB; ++rb) {
      for (int c0 = 0; c0 < Lp; c0 += kCommitChunk) {
        const int n = min(kCommitChunk, Lp - c0);
        __syncthreads();   // the previous chunk is fully consumed
        stage(c0, n);
        replay(One{}, rb, rb % NBUF, n);
      }
      store_block(rb, sb[rb % NBUF]);
      if (rb + NBUF < NB) load_block(rb + NBUF, sb[rb % NBUF]);
    }
  }
  TL_TRACE_POINT(a, 5);
}

// SPLIT workgroups per (request, v-head) slot of one layer.
template <int MODE, int D, bool F32IN, int SPLIT>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4))) void commit_kernel(CommitArgs a) {
  const int slot = blockIdx.x / SPLIT, part = blockIdx.x % SPLIT;
  commit_unit<MODE, D, F32IN, false, SPLIT>(a.c, a.ly, a.path_offsets, a.path, nullptr, slot / a.c.Hv,
                                            slot % a.c.Hv, part);
}

// Workgroups per slot in the unified commit: the delta rule's slots go to two
// (each holds its two row blocks and replays them side by side, as the
// single-layer commit does below its slot count threshold).
template <int MODE, int D>
constexpr int layers_split() {
  return (MODE == TL_MODE_GDN && CommitShape<D, MODE>::NRB % 2 == 0) ? 2 : 1;
}

// layers_split() workgroups per (layer, request, v-head) slot; consecutive
// workgroups walk the slot's parts, the v-heads, then the requests, then the
// layers.
template <int MODE, int D, bool F32IN, int NL>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4))) void commit_layers_kernel(
    CommitLayersArgsN<NL> a) {
  constexpr int SPLIT = layers_split<MODE, D>();
  const int per_layer = a.c.batch * a.c.Hv * SPLIT;
  const int layer = blockIdx.x / per_layer, rem = blockIdx.x % per_layer;
  const int slot = rem / SPLIT, part = rem % SPLIT;
  // a launch of one layer indexes its table statically, so that the kernel
  // arguments are read in a few wide loads at the start
  commit_unit<MODE, D, F32IN, true, SPLIT>(a.c, a.ly[NL == 1 ? 0 : layer], nullptr, nullptr, a.terminal,
                                           slot / a.c.Hv, slot % a.c.Hv, part);
}

// Accepted path of every request from its terminal node: path_len[b] and the
// path's request-local nodes, root first, at path[node_offsets[b] + t].  One
// workgroup per request.
__global__ __launch_bounds__(kThreads) void accepted_path_kernel(PathArgs a) {
  __shared__ int s_par[kMaxNodes];
  __shared__ int s_path[kMaxNodes];
  __shared__ int s_red[kWaves];
  const int tid = threadIdx.x, b = blockIdx.x;
  Request rq;
  if (!load_request(a.node_offsets, b, a.max_nodes, a.dev_err, rq)) return;
  const int T = rq.T, term = a.terminal[b];
  if (T == 0) {
    if (tid == 0) {
      if (term == -1) a.path_len[b] = 0;
      else report(a.dev_err, TL_EBADPATH);
    }
    return;
  }
  const int par = a.parent[rq.off + min(tid, T - 1)];
  if (tid < T) s_par[tid] = par;
  if (block_or_lds(tid < T && !(par == -1 || (par >= 0 && par < tid)), s_red)) {
    if (tid == 0) report(a.dev_err, TL_EBADTREE);
    return;
  }
  if (term < -1 || term >= T) {
    if (tid == 0) report(a.dev_err, TL_EBADPATH);
    return;
  }
  const int L = term < 0 ? 0 : path_to_root(term, s_par, s_path);
  if (tid == 0) a.path_len[b] = L;
  if (tid < L) a.path[rq.off + tid] = s_path[tid];
}

// Workgroups of the commit kernels that one GPU holds at once (four per
// compute unit: 128 registers and 35 KB of LDS each).
static long resident_commit_blocks() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  return 4L * cus;
}

template <int MODE, int D, bool F32IN, int SPLIT>
static tl_status launch_split(const CommitArgs& a, long slots, hipStream_t stream) {
  const long blocks = slots * SPLIT;
  if (blocks > 0x7fffffffL) return TL_EINVAL;
  hipLaunchKernelGGL((commit_kernel<MODE, D, F32IN, SPLIT>), dim3((unsigned)blocks), dim3(kThreads), 0,
                     stream, a);
  return hipGetLastError() == hipSuccess ? TL_OK : TL_EHIP;
}

// Fewer slots than the GPU holds workgroups at once: each slot's row blocks
// are spread over 2 or 4 workgroups (the replay is a chain of dependent
// steps per row block, so more of them run side by side).
template <int MODE, int D, bool F32IN>
static tl_status launch_one(const CommitArgs& a, hipStream_t stream) {
  const long slots = (long)a.c.batch * a.c.Hv;
  if (slots == 0) return TL_OK;
  constexpr int NRB = CommitShape<D, MODE>::NRB;
  const long resident = resident_commit_blocks();
  if constexpr (NRB % 4 == 0) {
    if (resident > 0 && 2 * slots < resident) return launch_split<MODE, D, F32IN, 4>(a, slots, stream);
  }
  if constexpr (NRB % 2 == 0) {
    if (resident > 0 && slots < resident) return launch_split<MODE, D, F32IN, 2>(a, slots, stream);
  }
  return launch_split<MODE, D, F32IN, 1>(a, slots, stream);
}

template <int MODE, int D, bool F32IN, int NL>
static tl_status launch_one(const CommitLayersArgsN<NL>& a, hipStream_t stream) {
  const long blocks = (long)a.num_layers * a.c.batch * a.c.Hv * layers_split<MODE, D>();
  if (blocks == 0) return TL_OK;
  if (blocks > 0x7fffffffL) return TL_EINVAL;
  hipLaunchKernelGGL((commit_layers_kernel<MODE, D, F32IN, NL>), dim3((unsigned)blocks), dim3(kThreads),
                     0, stream, a);
  return hipGetLastError() == hipSuccess ? TL_OK : TL_EHIP;
}

template <int MODE, bool F32IN, class Args>
static tl_status dispatch_d(int d, const Args& a, hipStream_t stream) {
  switch (d) {
    case 16: return launch_one<MODE, 16, F32IN>(a, stream);
    case 32: return launch_one<MODE, 32, F32IN>(a, stream);
    case 64: return launch_one<MODE, 64, F32IN>(a, stream);
    case 128: return launch_one<MODE, 128, F32IN>(a, stream);
    default: return TL_EUNSUPPORTED;
  }
}

template <class Args>
static tl_status dispatch(const tl_problem& p, const Args& a, hipStream_t stream) {
  if (p.mode == TL_MODE_GLA)
    return p.in_dtype == TL_F32 ? dispatch_d<TL_MODE_GLA, true>(p.d_k, a, stream)
                                : dispatch_d<TL_MODE_GLA, false>(p.d_k, a, stream);
  return p.in_dtype == TL_F32 ? dispatch_d<TL_MODE_GDN, true>(p.d_k, a, stream)
                              : dispatch_d<TL_MODE_GDN, false>(p.d_k, a, stream);
}

tl_status launch_commit(const tl_problem& p, const CommitArgs& a, hipStream_t stream) {
  return dispatch(p, a, stream);
}

// A layer whose slots alone fill the GPU goes out as a launch of its own:
// each launch then reads its states and writes them back in two broad
// phases, which on HBM3E outran one launch in which layers overlap and reads
// and writes mix.  Smaller layers share one launch, which keeps the GPU full.
tl_status launch_commit_layers(const tl_problem& p, const CommitLayersArgs& a, hipStream_t stream) {
  const long per_layer = (long)a.c.batch * a.c.Hv;
  const long resident = resident_commit_blocks();
  if (a.num_layers == 1 || resident == 0 || per_layer < resident) return dispatch(p, a, stream);
  CommitLayersArgsN<1> one;
  one.c = a.c;
  one.terminal = a.terminal;
  one.num_layers = 1;
  for (int l = 0; l < a.num_layers; ++l) {
    one.ly[0] = a.ly[l];
    const tl_status st = dispatch(p, one, stream);
    if (st != TL_OK) return st;
  }
  return TL_OK;
}

tl_status launch_accepted_path(const PathArgs& a, hipStream_t stream) {
  if (a.batch == 0) return TL_OK;
  hipLaunchKernelGGL(accepted_path_kernel, dim3((unsigned)a.batch), dim3(kThreads), 0, stream, a);
  return hipGetLastError() == hipSuccess ? TL_OK : TL_EHIP;
}

}  // namespace tl
