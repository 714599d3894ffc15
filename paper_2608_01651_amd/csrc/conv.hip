// Tree-parallel convolution front end (§4.3, Stage 1; §2.1) and the commit
// of the convolution state.
//
// A gated linear-attention layer forms q, k, v with a short causal depthwise
// convolution of its mixed projection x = [q | k | v] (C channels), then bias
// and SiLU; q and k are normalised per head, and the gates are prepared from
// their own projections.  On a token sequence the convolution reads the
// width - 1 preceding inputs; for a tree node those are its nearest
// ancestors on the root path, and above the root the window continues into
// the request's committed convolution state (the last width - 1 inputs of
// the prefix, oldest first).  Each node therefore depends only on a fixed
// number of ancestors: all nodes run at once, whatever the depth.
//
//   y_i[c] = bias[c] + sum_p W[c, p] s_i[p][c]    (s_i: window of node i,
//                                                  p = width - 1 is i itself)
//   z = y * sigmoid(y);  q, k: z / sqrt(sum_head z^2 + eps)
//   g = -exp(A_log[h]) * softplus(a + dt_bias[h]),  beta = sigmoid(b)
//
// conv_gates_kernel: one workgroup per (request, channel tile of 128).  In
// one round trip it copies the tile's rows of every node of the request and
// of the committed state straight into LDS (coalesced direct copies), and
// loads the parents (checked as a whole) and the gate inputs; the lane's
// weights were requested before that.  Every window is then read from LDS,
// so each node row crosses HBM once.  A tile row is CT / 8 lanes of 16
// bytes, and a wave takes 64 / (CT / 8) nodes at a time.
//
// conv_state_commit_kernel: one workgroup per (request, channel tile): the
// new state is the last width - 1 rows of (old state, accepted path rows),
// gathered into registers before the slot is overwritten.
#include <hip/hip_runtime.h>

#include "tl_device.h"
#include "tl_kernels.h"

namespace tl {

static_assert(kConvCommitTile == kThreads * 8, "one 8-channel chunk per thread");

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// log2(e) SiLU(y) from t = log2(e) y: t / (1 + 2^-t) = log2(e) y sigma(y).
// The convolution forms t directly (weights and bias scaled by log2(e) once),
// which saves a multiply per element; the factor log2(e) then cancels in the
// q/k normalisation (with eps scaled by log2(e)^2) and is taken out of v by
// the output scale.  Hardware exp2 and reciprocal (about 1 ulp each): the
// result is stored as bf16, 2^-8 relative, so their error is far below it.
// Large negative t gives exp2 = inf and rcp = 0, i.e. -0.
__device__ inline float silu_log2e(float t) {
  return t * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-t));
}
__device__ inline float softplus(float x) { return fmaxf(x, 0.f) + log1pf(expf(-fabsf(x))); }
__device__ inline float sigmoidf(float x) { return 1.f / (1.f + expf(-x)); }

template <int WIDTH, bool GDN, int CT>
__global__ __launch_bounds__(kThreads) void conv_gates_kernel(ConvArgs a) {
  static_assert(CT % 8 == 0 && 64 % (CT / 8) == 0, "a node row is a whole lane group");
  constexpr int LPN = CT / 8;               // lanes per node row of the tile (one 16-byte chunk each)
  constexpr int NPW = 64 / LPN;             // nodes per wave and pass
  constexpr int RB = CT * 2;                // bytes of a tile row
  constexpr int CSR = (WIDTH - 1 + NPW - 1) / NPW * NPW;   // state rows in LDS (whole copy instructions)
  extern __shared__ __align__(16) unsigned char conv_lds[];
  int* s_par = reinterpret_cast<int*>(conv_lds);                               // [kMaxNodes]
  __bf16* s_cs = reinterpret_cast<__bf16*>(conv_lds + kMaxNodes * 4);          // [CSR][tile]
  __bf16* s_x = s_cs + CSR * CT;                                               // [max_nodes rounded to NPW][tile]
  const int tile = blockIdx.x % a.tiles, b = blockIdx.x / a.tiles;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int C = a.C;
  TL_TRACE_POINT(a, 0);
  const int c0 = tile * CT + (lane % LPN) * 8;
  const bool live = c0 < C;
  const int cc = live ? c0 : C - 8;   // dead lanes read a valid chunk and store nothing

  // the lane's weights and bias (independent of the request: requested first)
  f32x4 wr[2 * WIDTH];
  {
    const f32x4* wv = reinterpret_cast<const f32x4*>(a.conv_weight + (size_t)cc * WIDTH);
#pragma unroll
    for (int t = 0; t < 2 * WIDTH; ++t) wr[t] = wv[t];
  }
  f32x4 b0 = *reinterpret_cast<const f32x4*>(a.conv_bias + cc);
  f32x4 b1 = *reinterpret_cast<const f32x4*>(a.conv_bias + cc + 4);

  // the slot is read with the node range (independent loads, one round trip)
  const int sidx = a.slot ? a.slot[b] : b;
  Request rq;
  if (!load_request(a.node_offsets, b, a.max_nodes, a.dev_err, rq)) return;
  const int T = rq.T;
  if (T == 0) return;
  if (sidx < 0 || sidx >= a.num_slots) {
    if (tid == 0) report(a.dev_err, TL_EINVAL);
    return;
  }

  // one round trip: the parents, the tile's rows of every node and of the
  // committed state (direct copies into LDS: 4 rows per wave instruction;
  // rows of dead channels copy a valid chunk), and the gate inputs
  const int par = tid < T ? a.parent[rq.off + tid] : -1;
  {
    const char* xg = reinterpret_cast<const char*>(reinterpret_cast<const __bf16*>(a.x) + cc);
    for (int r0 = wave * NPW; r0 < T; r0 += kWaves * NPW) {
      const int r = min(r0 + lane / LPN, T - 1);
      copy16_to_lds_async<true>(xg + (size_t)(rq.off + r) * C * 2, s_x + r0 * CT);   // read once
    }
    const char* cg = reinterpret_cast<const char*>(reinterpret_cast<const __bf16*>(a.conv_state) +
                                                   (size_t)sidx * (WIDTH - 1) * C + cc);
    if (wave == kWaves - 1) {
      for (int r0 = 0; r0 < CSR; r0 += NPW) {
        const int r = min(r0 + lane / LPN, WIDTH - 2);
        copy16_to_lds_async(cg + (size_t)r * C * 2, s_cs + r0 * CT);
      }
    }
  }
  // gates: the request's T * Hv of them, spread over all its tiles
  const int gx = tile * kThreads + tid;
  const bool has_gate = gx < T * a.Hv;
  const size_t gi = (size_t)rq.off * a.Hv + (has_gate ? gx : 0);
  const float ga = a.gate_a[gi];
  float gb = 0.f;
  if constexpr (GDN) gb = a.gate_b[gi];
  const int gh = (has_gate ? gx : 0) % a.Hv;
  const float alog = a.A_log[gh], dtb = a.dt_bias[gh];
  if (tid < T) s_par[tid] = par;
  wait_vmem();   // the direct copies (and everything else requested above)
  TL_TRACE_POINT(a, 1);
  if (__syncthreads_or(tid < T && !(par == -1 || (par >= 0 && par < tid)))) {
    if (tid == 0) report(a.dev_err, TL_EBADTREE);
    return;
  }
  if (has_gate) {
    a.g[gi] = -expf(alog) * softplus(ga + dtb);
    if constexpr (GDN) a.beta[gi] = sigmoidf(gb);
  }
  // gates beyond one per thread of the request's tiles (only when C / 16 < T Hv)
  for (int x = gx + a.tiles * kThreads; x < T * a.Hv; x += a.tiles * kThreads) {
    const size_t gj = (size_t)rq.off * a.Hv + x;
    const int h = x % a.Hv;
    a.g[gj] = -expf(a.A_log[h]) * softplus(a.gate_a[gj] + a.dt_bias[h]);
    if constexpr (GDN) a.beta[gj] = sigmoidf(a.gate_b[gj]);
  }

  const int nqk = a.Hk * a.dk;
  const bool norm = c0 < 2 * nqk;
  __bf16* dst0;
  size_t dst_row;
  if (c0 < nqk) {
    dst0 = reinterpret_cast<__bf16*>(a.q) + c0;
    dst_row = nqk;
  } else if (c0 < 2 * nqk) {
    dst0 = reinterpret_cast<__bf16*>(a.k) + (c0 - nqk);
    dst_row = nqk;
  } else {
    dst0 = reinterpret_cast<__bf16*>(a.v) + (c0 - 2 * nqk);
    dst_row = (size_t)a.Hv * a.dv;
  }
  const int lo = (lane % LPN) * 16;   // the lane's byte offset in a tile row
#pragma unroll
  for (int t = 0; t < 2 * WIDTH; ++t) wr[t] *= kLog2e;   // the convolution forms log2(e) y
  b0 *= kLog2e;
  b1 *= kLog2e;
  TL_TRACE_POINT(a, 2);

  for (int base = 0; base < T; base += kWaves * NPW) {
    const int n = base + wave * NPW + lane / LPN;
    const int nc = n < T ? n : T - 1;   // lanes past T compute a valid node and store nothing
    // window position WIDTH - 1 - s: the node s steps up, or, once the root
    // is passed, the committed state rows newest first.  j < 0 stands for
    // state row WIDTH - 1 + j, so a step is j <- parent(j) for a node and
    // j <- j - 1 past the root; the row is picked by a select, without
    // branches (lanes walk different paths)
    bf16x8 win[WIDTH];
    const char* xb = reinterpret_cast<const char*>(s_x) + lo;
    const char* cb = reinterpret_cast<const char*>(s_cs) + lo;
    win[WIDTH - 1] = *reinterpret_cast<const bf16x8*>(xb + nc * RB);
    int j = nc;
#pragma unroll
    for (int s = 1; s < WIDTH; ++s) {
      const int pj = s_par[j > 0 ? j : 0];
      j = j >= 0 ? pj : j - 1;
      const char* row = j >= 0 ? xb + j * RB : cb + (WIDTH - 1 + j) * RB;
      win[WIDTH - 1 - s] = *reinterpret_cast<const bf16x8*>(row);
    }
    float z[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float y = e < 4 ? b0[e] : b1[e - 4];
#pragma unroll
      for (int p = 0; p < WIDTH; ++p) {
        const int f = e * WIDTH + p;   // W[c0 + e, p]
        y += wr[f >> 2][f & 3] * (float)win[p][e];
      }
      z[e] = silu_log2e(y);   // log2(e) SiLU(y)
    }
    // per-head normalisation of q and k: a head's d_k channels are d_k / 8
    // adjacent lanes of one node's lane group
    float ss = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += z[e] * z[e];
    switch (a.dk) {   // uniform
      case 16: ss = group_sum<2>(ss); break;
      case 32: ss = group_sum<4>(ss); break;
      case 64: ss = group_sum<8>(ss); break;
      default: ss = group_sum<16>(ss); break;
    }
    const float scale = norm ? rsqrtf(ss + a.eps * (kLog2e * kLog2e)) : kLn2;
    if (live && n < T) {
      bf16x8 out;
#pragma unroll
      for (int e = 0; e < 8; ++e) out[e] = (__bf16)(z[e] * scale);
      __builtin_nontemporal_store(out, reinterpret_cast<bf16x8*>(dst0 + (size_t)(rq.off + n) * dst_row));
    }
  }
  TL_TRACE_POINT(a, 3);
}

// Channel tile of conv_gates.  Wider tiles (256, 512 channels: more bytes
// per round trip, fewer workgroups per CU) measured slower at the
// production and delta-rule shapes.
constexpr int kConvTileCh = 128;

static int conv_lds_bytes(int width, int max_nodes, int ct) {
  const int npw = 64 / (ct / 8);
  const int csr = (width - 1 + npw - 1) / npw * npw;
  return kMaxNodes * 4 + (csr + (max_nodes + npw - 1) / npw * npw) * ct * 2;
}

template <int WIDTH>
__global__ __launch_bounds__(kThreads) void conv_state_commit_kernel(ConvCommitArgs a) {
  __shared__ int s_par[kMaxNodes];
  const int tile = blockIdx.x % a.tiles, b = blockIdx.x / a.tiles;
  const int tid = threadIdx.x;
  // the terminal node and the slot are read with the node range (independent
  // loads, one round trip)
  const int term = a.terminal[b];
  const int sidx = a.slot ? a.slot[b] : b;
  Request rq;
  if (!load_request(a.node_offsets, b, a.max_nodes, a.dev_err, rq)) return;
  const int T = rq.T;
  if (sidx < 0 || sidx >= a.num_slots) {
    if (tid == 0) report(a.dev_err, TL_EINVAL);
    return;
  }
  // the whole forest is checked, as the recurrent-state commit does
  const int par = tid < T ? a.parent[rq.off + tid] : -1;
  if (tid < T) s_par[tid] = par;
  if (__syncthreads_or(tid < T && !(par == -1 || (par >= 0 && par < tid)))) {
    if (tid == 0) report(a.dev_err, TL_EBADTREE);
    return;
  }
  if (term < -1 || term >= T) {
    if (tid == 0) report(a.dev_err, TL_EBADPATH);
    return;
  }
  if (term < 0) return;
  const int C = a.C;
  const int c0 = tile * kConvCommitTile + tid * 8;
  if (c0 >= C) return;   // no barrier follows
  const __bf16* X = reinterpret_cast<const __bf16*>(a.x);
  __bf16* CS = reinterpret_cast<__bf16*>(a.conv_state) + (size_t)sidx * (WIDTH - 1) * C + c0;
  // new row q (oldest first) is the node s = WIDTH - 2 - q steps above the
  // terminal, or, once the root is passed after L nodes, old row q + L
  bf16x8 nr[WIDTH - 1];
  int j = term, L = 0;
#pragma unroll
  for (int s = 0; s < WIDTH - 1; ++s) {
    const int q = WIDTH - 2 - s;
    if (L == 0 && j < 0) L = s;
    if (L == 0) {
      nr[q] = *reinterpret_cast<const bf16x8*>(X + (size_t)(rq.off + j) * C + c0);
      j = s_par[j];
    } else {
      nr[q] = *reinterpret_cast<const bf16x8*>(CS + (size_t)(q + L) * C);
    }
  }
#pragma unroll
  for (int q = 0; q < WIDTH - 1; ++q) *reinterpret_cast<bf16x8*>(CS + (size_t)q * C) = nr[q];
}

template <int WIDTH, int CT>
static tl_status launch_conv_ct(ConvArgs a, bool gdn, hipStream_t stream) {
  a.tiles = (a.C + CT - 1) / CT;
  const long blocks = (long)a.batch * a.tiles;
  if (blocks == 0) return TL_OK;
  if (blocks > 0x7fffffffL) return TL_EINVAL;
  const int lds = conv_lds_bytes(WIDTH, a.max_nodes, CT);
  const void* k = gdn ? reinterpret_cast<const void*>(conv_gates_kernel<WIDTH, true, CT>)
                      : reinterpret_cast<const void*>(conv_gates_kernel<WIDTH, false, CT>);
  if (lds > 64 * 1024 &&
      hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, lds) != hipSuccess)
    return TL_EHIP;
  if (gdn)
    hipLaunchKernelGGL((conv_gates_kernel<WIDTH, true, CT>), dim3((unsigned)blocks), dim3(kThreads), lds, stream, a);
  else
    hipLaunchKernelGGL((conv_gates_kernel<WIDTH, false, CT>), dim3((unsigned)blocks), dim3(kThreads), lds, stream, a);
  return hipGetLastError() == hipSuccess ? TL_OK : TL_EHIP;
}

template <int WIDTH>
static tl_status launch_conv_w(const ConvArgs& a, bool gdn, hipStream_t stream) {
  return launch_conv_ct<WIDTH, kConvTileCh>(a, gdn, stream);
}

tl_status launch_conv_gates(const ConvArgs& a, int width, bool gdn, hipStream_t stream) {
  switch (width) {
    case 2: return launch_conv_w<2>(a, gdn, stream);
    case 3: return launch_conv_w<3>(a, gdn, stream);
    case 4: return launch_conv_w<4>(a, gdn, stream);
    default: return TL_EUNSUPPORTED;
  }
}

template <int WIDTH>
static tl_status launch_conv_commit_w(const ConvCommitArgs& a, hipStream_t stream) {
  const long blocks = (long)a.batch * a.tiles;
  if (blocks == 0) return TL_OK;
  if (blocks > 0x7fffffffL) return TL_EINVAL;
  hipLaunchKernelGGL((conv_state_commit_kernel<WIDTH>), dim3((unsigned)blocks), dim3(kThreads), 0, stream, a);
  return hipGetLastError() == hipSuccess ? TL_OK : TL_EHIP;
}

tl_status launch_conv_state_commit(const ConvCommitArgs& a, int width, hipStream_t stream) {
  switch (width) {
    case 2: return launch_conv_commit_w<2>(a, stream);
    case 3: return launch_conv_commit_w<3>(a, stream);
    case 4: return launch_conv_commit_w<4>(a, stream);
    default: return TL_EUNSUPPORTED;
  }
}

}  // namespace tl
