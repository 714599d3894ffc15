// Batch-wide verification-budget allocation and forest materialiser
// (§5.1 "Batch-wide utility allocation", §5.2 "CUDA Graph-native
// packed-forest execution").
//
// Each request brings a drafter's candidate tree (parents before children)
// with p(u | parent(u)) per node.  A node's utility rho(v) is the product of
// those probabilities along its root path.  Every root is kept; what the
// capacity leaves goes to the highest-rho candidates of the whole batch
// (ties: the lower batch-wide index first, so a parent always precedes its
// child and every request's selection stays prefix-connected), with at most
// max_nodes nodes per request.  A segmented count gives each request's
// budget, and the survivors are packed request by request, in candidate
// order, into the flat forest that verification takes.
//
// Two launches of fixed shape (a round can be captured once and replayed):
//  1. rho_rank_kernel, up to 16 workgroups of 1024 per request (about 512
//     in all), one candidate per thread: rho in fp32, root first, one
//     rounding per step (Jacobi sweeps in LDS: after k sweeps every node of
//     depth < k holds its final value), then each non-root candidate's rank
//     in its request's order: the number of (rho, index) keys above its own,
//     read by broadcast from LDS.  Each workgroup ranks one band of the
//     request's candidates, its waves splitting the keys.  The request's
//     eligible candidates (ranks below e_b = min(max_nodes, M_b) - roots) go
//     to the workspace in rank order, as rho bits and local indices with
//     their parents, next to its roots and its counts.
//  2. select_pack_kernel, one workgroup of 1024:
//     - the eligible lists, each already sorted, are copied to LDS;
//     - a radix selection (11, 11 and 9 bits) finds the rho t of the K-th best
//       eligible candidate (K = the capacity left after the roots) and how
//       many candidates with rho exactly t are still to be taken; on sorted
//       lists equal digits sit in runs, so each run adds its length to the
//       histogram with one LDS atomic, and one wave scans the bins;
//     - per request, binary searches count its keys above t and equal to t;
//       the ties go to the lowest batch-wide indices, i.e. to requests in
//       batch order; budget = roots + taken, and a scan gives node_offsets;
//     - packing: the selected nodes are the roots and the `budget - roots`
//       first entries of the request's list (always a prefix-connected set);
//       each sets its bit in a bitmap over the batch's candidates, and in
//       batch order a node's packed row is the number of set bits before it
//       (a scan over the bitmap's words); parents are renumbered the same way.
//     Only the eligible and the selected candidates are touched here.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>

#include "tl_device.h"
#include "tl_kernels.h"

// The workspace of tree_budget_select_noalloc: one copy per GPU, held until
// the process ends.  In host code `scratch` names a host-side stand-in, not
// device memory: only the address hipGetSymbolAddress returns for the
// current device may be handed to kernels or copies.
static __device__ __align__(256) unsigned char scratch[tl::kBudgetScratchBytes];

namespace tl {

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};   // device address of `scratch`, per device
}  // namespace

// Device address of the current device's copy of `scratch`: looked up once
// per device, with that device current, and kept.
tl_status budget_scratch(void** ptr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return TL_EHIP;
  if (dev < 0 || dev >= kMaxDevices) return TL_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return TL_EHIP;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return TL_OK;
}

namespace {

constexpr int kRankThreads = kBudgetMaxTree;          // launch 1: one candidate per thread
constexpr int kRankWaves = kRankThreads / 64;
constexpr int kRankBlocks = 512;                        // launch 1: target workgroups
constexpr int kSelWaves = kSelectThreads / 64;
constexpr int kBins = 2048;                            // widest radix digit: 11 bits
constexpr int kNotEligible = 0x7fffffff;              // rank of a rejected request's non-roots


// A request's candidate range is usable when it lies inside the arrays and
// fits the per-request bound; the second launch rejects the batch otherwise.
__device__ inline bool range_ok(int o0, int o1, int num_candidates) {
  return o0 >= 0 && o1 >= o0 && o1 <= num_candidates && o1 - o0 <= kBudgetMaxTree;
}

__device__ inline int lane_id() { return (int)(threadIdx.x & 63); }

// Cross-lane moves by DPP (no LDS round trip).  `dpp<CTRL, ROWS>` reads the
// source lane CTRL names; lanes without one, and rows outside the ROWS mask,
// read 0.  Every lane of the wave must be active.
template <int CTRL, int ROWS = 0xF>
__device__ inline int dpp(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, ROWS, 0xF, true);
}
constexpr int kRowShr1 = 0x111, kRowShr2 = 0x112, kRowShr4 = 0x114, kRowShr8 = 0x118;
constexpr int kRowBcast15 = 0x142, kRowBcast31 = 0x143, kWaveShr1 = 0x138;

// Inclusive scan over the 64 lanes: within each row of 16 lanes by shifts of
// 1, 2, 4 and 8, then each row's total into the rows above it (lane 15 of a
// row into the next row, lane 31 into rows 2 and 3).
__device__ inline int wave_inclusive_scan(int x) {
  x += dpp<kRowShr1>(x);
  x += dpp<kRowShr2>(x);
  x += dpp<kRowShr4>(x);
  x += dpp<kRowShr8>(x);
  x += dpp<kRowBcast15, 0xA>(x);
  x += dpp<kRowBcast31, 0xC>(x);
  return x;
}

// Sum over the 64 lanes, the same in every lane.
__device__ inline int wave_sum(int x) {
  return __builtin_amdgcn_readlane(wave_inclusive_scan(x), 63);
}

// The value of the lane below (0 in lane 0).
__device__ inline int lane_below(int x) { return dpp<kWaveShr1>(x); }

// Sum over the workgroup (s_part: one int per wave).
template <int NW>
__device__ inline int block_sum(int x, int* s_part) {
  x = wave_sum(x);
  if (lane_id() == 0) s_part[threadIdx.x >> 6] = x;
  __syncthreads();
  int t = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) t += s_part[w];
  __syncthreads();
  return t;
}

// Inclusive scan of one value per thread over the workgroup; *total gets the sum.
template <int NW>
__device__ inline int block_inclusive_scan(int x, int* s_part, int* total) {
  const int wave = threadIdx.x >> 6;
  x = wave_inclusive_scan(x);
  if (lane_id() == 63) s_part[wave] = x;
  __syncthreads();
  int add = 0, t = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    add += w < wave ? s_part[w] : 0;
    t += s_part[w];
  }
  __syncthreads();
  *total = t;
  return x + add;
}

// Sort key of a non-root candidate: rho's magnitude bits above, the
// complemented request-local index below; larger key = earlier in the order.
// Every such key exceeds 0, the key of roots and of the padding.
__device__ inline uint64_t order_key(float rho, int v) {
  return ((uint64_t)(__float_as_uint(rho) & 0x7fffffffu) << 32) | (uint64_t)(0xffffffffu - (uint32_t)v);
}

// Number of leading keys of the descending list L[0..n) that are > t
// (STRICT false) or >= t (STRICT true).
template <bool STRICT>
__device__ inline int count_above(const uint32_t* L, int n, uint32_t t) {
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (STRICT ? L[mid] >= t : L[mid] > t) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

}  // namespace

// ---------------------------------------------------------------------------
// 1. rho and ranks
// ---------------------------------------------------------------------------
// Launch 1 runs `slices` workgroups per request (block = request * slices +
// slice).  Every one of them loads the whole tree and computes every rho (the
// sweep needs all of them), then ranks only its own band of candidates, with
// the 16 waves splitting the keys of the request between them; slice 0 also
// writes the request's roots and meta entries.
__global__ __launch_bounds__(kRankThreads) void rho_rank_kernel(BudgetArgs a) {
  __shared__ float s_rho[2][kBudgetMaxTree];
  __shared__ __align__(16) uint64_t s_key[kBudgetMaxTree + 8];
  __shared__ int s_cnt[kBudgetMaxTree];
  __shared__ int s_part[kRankWaves];
  const int slices = (int)gridDim.x / a.batch;
  const int b = (int)blockIdx.x / slices, s = (int)blockIdx.x - b * slices, v = threadIdx.x;
  const int lane = v & 63, wave = v >> 6;
  const int o0 = a.cand_offsets[b], o1 = a.cand_offsets[b + 1];
  if (!range_ok(o0, o1, a.num_candidates)) return;   // the second launch reports it
  const int M = o1 - o0;
  // this slice's band [c0, c1): bands of a multiple of 64 candidates
  const int C = max(64, ((M + slices - 1) / slices + 63) & ~63);
  const int c0 = s * C, c1 = min(M, c0 + C);
  if (s > 0 && c0 >= c1) return;   // an empty band (slice 0 always runs)
  const bool mine_band = v >= c0 && v < c1;
  TL_TRACE_POINT(a, 0);
  int p = -2, tree_bad = 0, prob_bad = 0;
  float pr = 0.f;
  if (v < M) {
    p = a.cand_parent[o0 + v];
    pr = a.cand_prob[o0 + v];
    s_rho[0][v] = pr;
    tree_bad = !(p == -1 || (p >= 0 && p < v));
    prob_bad = !(pr >= 0.f && pr <= 1.f);   // NaN fails too
  }
  const int mn = a.max_nodes;
  int roots;
  if (s == 0) {   // roots: their count, and their indices in order into the workspace
    const int rix = block_inclusive_scan<kRankWaves>(p == -1, s_part, &roots) - (p == -1);
    if (p == -1 && rix < mn) a.ws_root[(size_t)b * mn + rix] = (uint16_t)v;
  } else {
    roots = __syncthreads_count(p == -1);
  }
  const bool any_tree_bad = __syncthreads_or(tree_bad), any_prob_bad = __syncthreads_or(prob_bad);
  TL_TRACE_POINT(a, 1);
  const bool rejected = any_tree_bad || any_prob_bad;
  // eligible candidates: ranks below min(max_nodes, M) - roots (none if rejected)
  const int elig = rejected ? 0 : max(0, min(mn, M) - roots);
  if (s == 0 && v == 0) {
    a.ws_meta[4 * b] = roots;
    a.ws_meta[4 * b + 1] = elig;
    a.ws_meta[4 * b + 2] = rejected;
  }
  if (rejected) {
    // the request keeps its roots and nothing else
    if (s == 0 && v == 0) report(a.dev_err, any_tree_bad ? TL_EBADTREE : TL_EINVAL);
    if (mine_band) {
      a.rho[o0 + v] = 0.f;
      a.rank[o0 + v] = p == -1 ? -1 : kNotEligible;
    }
    return;
  }
  // rho(v) = rho(parent) * p(v), one fp32 rounding per step, root first
  int cur = 0;
  for (;;) {
    int changed = 0;
    if (v < M) {
      const float r = p < 0 ? pr : s_rho[cur][p] * pr;
      s_rho[cur ^ 1][v] = r;
      changed = __float_as_uint(r) != __float_as_uint(s_rho[cur][v]);
    }
    cur ^= 1;
    if (!__syncthreads_or(changed)) break;
  }
  TL_TRACE_POINT(a, 2);
  const float rho = v < M ? s_rho[cur][v] : 0.f;
  s_key[v] = v < M && p >= 0 ? order_key(rho, v) : 0ull;   // zero for roots and past M
  if (v < 8) s_key[kBudgetMaxTree + v] = 0ull;
  if (v < C) s_cnt[v] = 0;
  __syncthreads();
  // rank = keys above mine (roots and padding have key 0: never above).
  // Work items: (64-candidate block of the band, part of the key range)
  {
    const int nblk = (c1 - c0 + 63) >> 6;          // 0 (an empty request) .. 16
    const int parts = nblk > 0 ? max(1, kRankWaves / nblk) : 1;
    const int M8 = (M + 7) & ~7;
    const int span = ((M8 / 8 + parts - 1) / parts) * 8;
    for (int it = wave; it < nblk * parts; it += kRankWaves) {   // uniform per wave
      const int blk = it % nblk, part = it / nblk;
      const int c = c0 + 64 * blk + lane;
      const uint64_t mine = c < c1 ? s_key[c] : ~0ull;   // past the band: counts nothing
      const int u0 = part * span, u1 = min(M8, u0 + span);
      int cnt = 0;
      for (int u = u0; u < u1; u += 8) {
        uint64_t k[8];
#pragma unroll
        for (int j = 0; j < 8; j += 2) {
          const ulonglong2 two = *reinterpret_cast<const ulonglong2*>(&s_key[u + j]);
          k[j] = two.x;
          k[j + 1] = two.y;
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) cnt += k[j] > mine;
      }
      if (c < c1) {
        if (parts == 1) s_cnt[c - c0] = cnt;
        else atomicAdd(&s_cnt[c - c0], cnt);
      }
    }
  }
  __syncthreads();
  if (mine_band) {
    const int cnt = s_cnt[v - c0];
    a.rho[o0 + v] = rho;
    a.rank[o0 + v] = p < 0 ? -1 : cnt;
    if (p >= 0 && cnt < elig) {   // the request's eligible list, in rank order
      a.ws_key[(size_t)b * mn + cnt] = __float_as_uint(rho) & 0x7fffffffu;
      a.ws_cand[(size_t)b * mn + cnt] = (uint32_t)v | (uint32_t)(p + 1) << 16;
    }
  }
  TL_TRACE_POINT(a, 3);
}

// ---------------------------------------------------------------------------
// 2. batch-wide selection, budgets, node_offsets and packing
// ---------------------------------------------------------------------------
// LDS of select_pack_kernel: the histogram, five per-request arrays, and a
// region that holds the sorted key lists during the selection and the
// candidates' selection bitmap with its word offsets during the packing.
__host__ __device__ inline int budget_region_words(int num_candidates) {
  const int words = (num_candidates + 31) / 32;
  return num_candidates > 2 * words ? num_candidates : 2 * words;
}

int budget_select_lds_bytes(int batch, int num_candidates) {
  return 4 * (kBins + (batch + 1) + 4 * batch + budget_region_words(num_candidates));
}

namespace {

// Wave 0, after a histogram pass: the bin that holds the krem-th largest
// active key (lane l owns bins l*PER .. l*PER+PER-1, read and cleared as int4).
template <int PER>
__device__ inline void pick_bin(int* s_hist, uint32_t prefix, int width, int krem, int* s_prefix,
                                int* s_krem) {
  const int lane = lane_id();
  int h[PER];
  int4* row = reinterpret_cast<int4*>(s_hist + lane * PER);
#pragma unroll
  for (int j = 0; j < PER / 4; ++j) {
    const int4 q = row[j];
    h[4 * j] = q.x;
    h[4 * j + 1] = q.y;
    h[4 * j + 2] = q.z;
    h[4 * j + 3] = q.w;
  }
  int tot = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j) tot += h[j];
  const int incl = wave_inclusive_scan(tot);
  int above = __builtin_amdgcn_readlane(incl, 63) - incl;   // the bins of the lanes above this one
#pragma unroll
  for (int j = PER - 1; j >= 0; --j) {
    if (above < krem && krem <= above + h[j]) {   // exactly one bin satisfies this
      *s_prefix = (int)((prefix << width) | (uint32_t)(lane * PER + j));
      *s_krem = krem - above;
    }
    above += h[j];
  }
#pragma unroll
  for (int j = 0; j < PER / 4; ++j) row[j] = make_int4(0, 0, 0, 0);
}

// One radix pass over the sorted lists s_key[0..E): each run of equal digits
// among the keys that match `prefix` adds its length to its bin.
__device__ inline void histogram_pass(const uint32_t* s_key, int E, int* s_hist, int shift, int width,
                                      bool first, uint32_t prefix) {
  const int lane = lane_id();
  const uint32_t dmask = (1u << width) - 1u;
  for (int base = (int)(threadIdx.x >> 6) * 64; base < E; base += kSelectThreads) {   // uniform per wave
    const int pos = base + lane;
    const uint32_t key = pos < E ? s_key[pos] : 0u;
    const bool act = pos < E && (first || (key >> (shift + width)) == prefix);
    const int digit = (int)((key >> shift) & dmask);
    const int prev_digit = lane_below(digit);
    const int prev_act = lane_below((int)act);
    const bool head = act && (lane == 0 || !prev_act || prev_digit != digit);
    const uint64_t stops = __ballot(head || !act);
    if (head) {   // the run of equal digits that starts here
      const uint64_t rest = lane == 63 ? 0ull : stops >> (lane + 1);
      const int len = rest ? __builtin_ctzll(rest) + 1 : 64 - lane;
      atomicAdd(&s_hist[digit], len);
    }
  }
}

}  // namespace

__global__ __launch_bounds__(kSelectThreads) void select_pack_kernel(BudgetArgs a) {
  extern __shared__ __align__(16) int s_dyn[];
  __shared__ int s_part[kSelWaves];
  __shared__ int s_flag, s_prefix, s_krem;
  const int B = a.batch, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, mn = a.max_nodes;
  constexpr int kGroup = 8;   // requests per wave whose lists or entries are in flight together
  int* s_hist = s_dyn;               // [kBins] (16-byte aligned: read as int4)
  int* s_offs = s_hist + kBins;      // [B + 1] candidate offsets
  int* s_roots = s_offs + B + 1;     // [B] roots
  int* s_elig = s_roots + B;         // [B] eligible candidates e_b, then taken ones
  int* s_base = s_elig + B;          // [B] start of the request's sorted list in s_key
  int* s_noff = s_base + B;          // [B] packed offset of the request
  uint32_t* s_key = reinterpret_cast<uint32_t*>(s_noff + B);        // the sorted lists, then ...
  uint32_t* s_bits = s_key;                                          // ... a bit per candidate
  int* s_wpre = reinterpret_cast<int*>(s_key) + (a.num_candidates + 31) / 32;   // and word offsets
  TL_TRACE_POINT(a, 8);

  // -- shape, roots, eligible counts (from the first launch) ---------------
  if (tid == 0) s_flag = 0;
  for (int b = tid; b <= B; b += kSelectThreads) s_offs[b] = a.cand_offsets[b];
  int r_in = 0, e_in = 0;
  if (tid < B) {
    r_in = a.ws_meta[4 * tid];
    e_in = a.ws_meta[4 * tid + 1];
  }
  for (int i = tid; i < kBins; i += kSelectThreads) s_hist[i] = 0;
  __syncthreads();
  int flags = 0, roots = 0, elig = 0;
  if (tid == 0) {
    flags |= s_offs[0] != 0;   // 1 = malformed offsets, 2 = a size or count out of range
    flags |= (s_offs[B] > a.num_candidates) << 1;
  }
  if (tid < B) {
    const int m = s_offs[tid + 1] - s_offs[tid];
    flags |= m < 0;
    flags |= (m > kBudgetMaxTree || r_in > mn) << 1;
    roots = r_in;
    elig = e_in;
    s_roots[tid] = roots;
    s_elig[tid] = elig;
  }
  if (flags) atomicOr(&s_flag, flags);
  roots = block_sum<kSelWaves>(roots, s_part);   // its barriers also publish s_flag
  int err = (s_flag & 1) ? TL_EBADTREE : s_flag ? TL_EINVAL : TL_OK;
  const int K = a.capacity - roots;   // non-root nodes the capacity leaves
  if (err == TL_OK && K < 0) err = TL_EINVAL;
  if (err != TL_OK) {   // nothing selected: every budget is zero
    if (tid == 0) report(a.dev_err, err);
    for (int b = tid; b <= B; b += kSelectThreads) a.node_offsets[b] = 0;
    return;
  }
  int E;
  const int ebase = block_inclusive_scan<kSelWaves>(elig, s_part, &E) - elig;
  if (tid < B) s_base[tid] = ebase;
  const int M = s_offs[B];
  __syncthreads();   // s_base
  TL_TRACE_POINT(a, 9);

  int take = 0;   // this thread's request (tid < B): candidates taken
  if (K > 0 && K < E) {
    // -- the eligible lists, already sorted, into LDS.  A list has at most
    // max_nodes <= 256 keys.  With a few requests per wave: direct copies of
    // 64 keys per wave instruction (no registers, every list in flight at
    // once, lanes past the list's end masked off).  With more, the direct
    // copies issue too slowly; a wave then loads eight requests' lists at
    // once (four 64-lane loads each) into registers and stores them.
    if (B <= 4 * kSelWaves) {
      for (int b = wave; b < B; b += kSelWaves) {   // uniform per wave
        const int n = s_elig[b];
        const uint32_t* src = a.ws_key + (size_t)b * mn;
        uint32_t* dst = s_key + s_base[b];
        for (int c = 0; c < n; c += 64)   // uniform
          if (c + lane < n) copy4_to_lds_async(src + c + lane, dst + c);
      }
      wait_vmem();   // the copies are not tracked by the compiler
    } else {
      for (int b0 = wave; b0 < B; b0 += kGroup * kSelWaves) {   // uniform per wave
        uint32_t t[kGroup][4];
#pragma unroll
        for (int g = 0; g < kGroup; ++g) {
          const int b = b0 + g * kSelWaves, n = b < B ? s_elig[b] : 0;
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const int r = lane + 64 * c;
            if (r < n) t[g][c] = a.ws_key[(size_t)b * mn + r];
          }
        }
#pragma unroll
        for (int g = 0; g < kGroup; ++g) {
          const int b = b0 + g * kSelWaves, n = b < B ? s_elig[b] : 0;
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const int r = lane + 64 * c;
            if (r < n) s_key[s_base[b] + r] = t[g][c];
          }
        }
      }
    }
    __syncthreads();
    TL_TRACE_POINT(a, 10);
    // -- radix selection of the K-th best key: 11, 11 and 9 bits -----------
    uint32_t prefix = 0;
    int krem = K;
    histogram_pass(s_key, E, s_hist, 20, 11, true, 0u);
    __syncthreads();
    if (wave == 0) pick_bin<32>(s_hist, prefix, 11, krem, &s_prefix, &s_krem);
    __syncthreads();
    prefix = (uint32_t)s_prefix;
    krem = s_krem;
    histogram_pass(s_key, E, s_hist, 9, 11, false, prefix);
    __syncthreads();
    if (wave == 0) pick_bin<32>(s_hist, prefix, 11, krem, &s_prefix, &s_krem);
    __syncthreads();
    prefix = (uint32_t)s_prefix;
    krem = s_krem;
    histogram_pass(s_key, E, s_hist, 0, 9, false, prefix);
    __syncthreads();
    if (wave == 0) pick_bin<8>(s_hist, prefix, 9, krem, &s_prefix, &s_krem);
    __syncthreads();
    prefix = (uint32_t)s_prefix;
    krem = s_krem;
    TL_TRACE_POINT(a, 11);
    // -- per request: keys above the threshold, and ties; ties in batch order
    int gt = 0, tie = 0;
    if (tid < B) {
      const uint32_t* L = s_key + s_base[tid];
      const int n = s_elig[tid];
      gt = count_above<false>(L, n, prefix);
      tie = count_above<true>(L, n, prefix) - gt;
    }
    int all_ties;
    const int before = block_inclusive_scan<kSelWaves>(tie, s_part, &all_ties) - tie;
    take = gt + min(max(krem - before, 0), tie);
  } else if (K >= E) {
    take = tid < B ? s_elig[tid] : 0;
  }
  // -- budgets and node_offsets (one request per thread) --------------------
  const int q = tid < B ? s_roots[tid] + take : 0;
  int total;
  const int incl = block_inclusive_scan<kSelWaves>(q, s_part, &total);
  if (tid < B) {
    a.node_offsets[tid + 1] = incl;
    s_noff[tid] = incl - q;
    s_elig[tid] = take;
  }
  if (tid == 0) a.node_offsets[0] = 0;
  const int words = (M + 31) / 32;
  for (int w = tid; w < words; w += kSelectThreads) s_bits[w] = 0u;   // the keys are dead
  __syncthreads();
  TL_TRACE_POINT(a, 12);

  // -- packing: a bit per selected candidate (the roots and the best-ranked
  // `take`, at most max_nodes <= 256 per request: four chunks of a wave); in
  // batch order a node's packed row is the number of selected candidates
  // before it, which a word scan of the bitmap gives.  A selected node's
  // entry is its index in the request with its parent + 1 above bit 16 (0 for
  // a root); up to kGroup * 16 requests the entries stay in registers between
  // the two passes
  using Entries = uint32_t[kGroup][4];
  auto load_entries = [&](int b0, Entries& e) __attribute__((always_inline)) {
#pragma unroll
    for (int g = 0; g < kGroup; ++g) {
      const int b = b0 + g * kSelWaves;
      const int nr = b < B ? s_roots[b] : 0, n = b < B ? nr + s_elig[b] : 0;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int j = lane + 64 * c;
        if (j < n) e[g][c] = j < nr ? (uint32_t)a.ws_root[(size_t)b * mn + j] : a.ws_cand[(size_t)b * mn + (j - nr)];
      }
    }
  };
  auto apply = [&](int b0, const Entries& e, auto&& fn) __attribute__((always_inline)) {
#pragma unroll
    for (int g = 0; g < kGroup; ++g) {
      const int b = b0 + g * kSelWaves;
      const int n = b < B ? s_roots[b] + s_elig[b] : 0;
#pragma unroll
      for (int c = 0; c < 4; ++c)
        if (lane + 64 * c < n) fn(b, s_offs[b], s_offs[b] + (int)(e[g][c] & 0xffffu), (int)(e[g][c] >> 16) - 1);
    }
  };
  const bool resident = B <= kGroup * kSelWaves;
  Entries kept;
  if (resident) load_entries(wave, kept);
  auto each_selected = [&](auto&& fn) __attribute__((always_inline)) {
    if (resident) {
      apply(wave, kept, fn);
    } else {
      for (int b0 = wave; b0 < B; b0 += kGroup * kSelWaves) {   // uniform per wave
        Entries e;
        load_entries(b0, e);
        apply(b0, e, fn);
      }
    }
  };
  each_selected([&](int, int, int i, int) { atomicOr(&s_bits[i >> 5], 1u << (i & 31)); });
  __syncthreads();
  {
    // word offsets: thread t scans words t * per .. t * per + per - 1
    const int per = (words + kSelectThreads - 1) / kSelectThreads;
    int cnt = 0;
    for (int w = tid * per; w < min(words, (tid + 1) * per); ++w) cnt += __popc(s_bits[w]);
    int all;
    int run = block_inclusive_scan<kSelWaves>(cnt, s_part, &all) - cnt;
    for (int w = tid * per; w < min(words, (tid + 1) * per); ++w) {
      s_wpre[w] = run;
      run += __popc(s_bits[w]);
    }
  }
  __syncthreads();
  TL_TRACE_POINT(a, 13);
  auto row_of = [&](int i) __attribute__((always_inline)) {
    return s_wpre[i >> 5] + __popc(s_bits[i >> 5] & ((1u << (i & 31)) - 1u));
  };
  int broken = 0;
  each_selected([&](int b, int o0, int i, int p) {
    const int k = row_of(i);
    const bool pin = p >= 0 && ((s_bits[(o0 + p) >> 5] >> ((o0 + p) & 31)) & 1u);
    broken |= (p != -1 && !pin) || k >= a.capacity;   // never for a consistent selection
    if (k < a.capacity) {
      a.src[k] = i;
      a.parent[k] = p == -1 ? -1 : (pin ? row_of(o0 + p) - s_noff[b] : -1);
    }
  });
  if (broken) report(a.dev_err, TL_EBADTREE);
  TL_TRACE_POINT(a, 15);
}

tl_status launch_budget_select(const BudgetArgs& a, hipStream_t stream) {
  if (a.batch == 0) return TL_OK;
  const int lds = budget_select_lds_bytes(a.batch, a.num_candidates);
  if (lds + 256 > 160 * 1024) return TL_EUNSUPPORTED;
  if (lds > 64 * 1024 &&
      hipFuncSetAttribute(reinterpret_cast<const void*>(select_pack_kernel),
                          hipFuncAttributeMaxDynamicSharedMemorySize, lds) != hipSuccess)
    return TL_EHIP;
  // launch 1: about kRankBlocks workgroups in all, at most one band of 64
  // candidates each
  const int slices = std::min(kBudgetMaxTree / 64, std::max(1, kRankBlocks / a.batch));
  hipLaunchKernelGGL(rho_rank_kernel, dim3((unsigned)(a.batch * slices)), dim3(kRankThreads), 0, stream, a);
  hipLaunchKernelGGL(select_pack_kernel, dim3(1), dim3(kSelectThreads), lds, stream, a);
  return hipGetLastError() == hipSuccess ? TL_OK : TL_EHIP;
}

}  // namespace tl
