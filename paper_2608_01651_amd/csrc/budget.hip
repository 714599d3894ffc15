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
//  1. rho_rank_kernel, one workgroup of 1024 per request, one candidate per
//     thread: rho in fp32, root first, one rounding per step (Jacobi sweeps
//     in LDS: after k sweeps every node of depth < k holds its final value),
//     then each non-root candidate's rank in its request's order: the number
//     of (rho, index) keys above its own, read by broadcast from LDS.  The
//     request's root count (negated minus one when the request is rejected)
//     goes to node_offsets[b + 1] for the second launch.
//  2. select_pack_kernel, one workgroup of 1024:
//     - a request's eligible candidates are its ranks below
//       e_b = min(max_nodes, M_b) - roots, so the eligible total E and every
//       request's place in a sorted key array follow from the offsets alone;
//     - one coalesced sweep scatters each eligible candidate's rho bits to
//       position base_b + rank: per request a descending list in LDS;
//     - a radix selection (11, 11 and 9 bits) finds the rho t of the K-th best
//       eligible candidate (K = the capacity left after the roots) and how
//       many candidates with rho exactly t are still to be taken; on sorted
//       lists equal digits sit in runs, so each run adds its length to the
//       histogram with one LDS atomic, and one wave scans the bins;
//     - per request, binary searches count its keys above t and equal to t;
//       the ties go to the lowest batch-wide indices, i.e. to requests in
//       batch order; budget = roots + taken, and a scan gives node_offsets;
//     - packing: the selected nodes are the roots and the `budget - roots`
//       best-ranked candidates (always such a prefix of the request's order);
//       in batch order, a node's packed row is the number of selected
//       candidates before it, so coalesced sweeps over contiguous per-wave
//       segments, ballots and one scan of the wave totals number them, and
//       parents are renumbered through LDS.
#include <hip/hip_runtime.h>

#include "tl_device.h"
#include "tl_kernels.h"

namespace tl {

namespace {

constexpr int kRankThreads = kBudgetMaxTree;          // launch 1: one candidate per thread
constexpr int kRankWaves = kRankThreads / 64;
constexpr int kSelWaves = kSelectThreads / 64;
constexpr int kBins = 2048;                            // widest radix digit: 11 bits
constexpr int kSegChunks = kBudgetMaxCandidates / (kSelWaves * 64);   // 64-candidate chunks per wave
constexpr int kNotEligible = 0x7fffffff;              // rank of a rejected request's non-roots

static_assert(kSegChunks <= 32, "a wave's selection bits must fit one 32-bit mask");

// A request's candidate range is usable when it lies inside the arrays and
// fits the per-request bound; the second launch rejects the batch otherwise.
__device__ inline bool range_ok(int o0, int o1, int num_candidates) {
  return o0 >= 0 && o1 >= o0 && o1 <= num_candidates && o1 - o0 <= kBudgetMaxTree;
}

__device__ inline int lane_id() { return (int)(threadIdx.x & 63); }

// lanes below this one whose bit is set in `mask`
__device__ inline int lanes_below(uint64_t mask) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ inline int wave_sum(int x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

__device__ inline int wave_inclusive_scan(int x) {
  const int lane = lane_id();
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  return x;
}

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

// The request of candidate i: the last b with s_offs[b] <= i (i < s_offs[B]).
__device__ inline int request_of(const int* s_offs, int B, int i) {
  int lo = 0, hi = B - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (s_offs[mid] <= i) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// Moves b forward to the request that holds candidate i (i increases).
__device__ inline int advance_request(const int* s_offs, int B, int b, int i) {
  while (b < B - 1 && s_offs[b + 1] <= i) ++b;
  return b;
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
__global__ __launch_bounds__(kRankThreads) void rho_rank_kernel(BudgetArgs a) {
  __shared__ float s_rho[2][kBudgetMaxTree];
  __shared__ __align__(16) uint64_t s_key[kBudgetMaxTree + 8];
  __shared__ int s_part[kRankWaves];
  const int b = blockIdx.x, v = threadIdx.x;
  const int o0 = a.cand_offsets[b], o1 = a.cand_offsets[b + 1];
  if (!range_ok(o0, o1, a.num_candidates)) return;   // the second launch reports it
  const int M = o1 - o0;
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
  const int roots = block_sum<kRankWaves>(p == -1, s_part);
  const bool any_tree_bad = __syncthreads_or(tree_bad), any_prob_bad = __syncthreads_or(prob_bad);
  TL_TRACE_POINT(a, 1);
  if (v == 0) a.node_offsets[b + 1] = (any_tree_bad || any_prob_bad) ? -(roots + 1) : roots;
  if (any_tree_bad || any_prob_bad) {
    // the request keeps its roots and nothing else
    if (v == 0) report(a.dev_err, any_tree_bad ? TL_EBADTREE : TL_EINVAL);
    if (v < M) {
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
  const uint64_t mine = v < M && p >= 0 ? order_key(rho, v) : 0ull;
  s_key[v] = mine;   // zero for roots and past M
  if (v < 8) s_key[kBudgetMaxTree + v] = 0ull;
  __syncthreads();
  if (v < M) {
    // rank = keys above mine (roots and padding have key 0: never above)
    int cnt = 0;
    const int M8 = (M + 7) & ~7;
    for (int u = 0; u < M8; u += 8) {
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
    a.rho[o0 + v] = rho;
    a.rank[o0 + v] = p < 0 ? -1 : cnt;
  }
  TL_TRACE_POINT(a, 3);
}

// ---------------------------------------------------------------------------
// 2. batch-wide selection, budgets, node_offsets and packing
// ---------------------------------------------------------------------------
int budget_select_lds_bytes(int batch, int num_candidates) {
  return 4 * (kBins + (batch + 1) + 4 * batch + num_candidates);
}

namespace {

// A lane's request while it walks its candidates in increasing order.
struct Cursor {
  int b, end;   // request b holds candidates up to end - 1
  __device__ void seek(const int* s_offs, int B, int i) {
    b = request_of(s_offs, B, i);
    end = s_offs[b + 1];
  }
  // Moves to the request of candidate i (i never decreases); true if it changed.
  __device__ bool advance(const int* s_offs, int B, int i) {
    if (i < end) return false;
    do {
      ++b;
      end = s_offs[b + 1];
    } while (b < B - 1 && end <= i);
    return true;
  }
};

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
  int t = tot;   // inclusive suffix over lanes >= this one
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_down(t, o, 64);
    if (lane + o < 64) t += y;
  }
  int above = t - tot;
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
    const int prev_digit = __shfl_up(digit, 1, 64);
    const int prev_act = __shfl_up((int)act, 1, 64);
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
  const int B = a.batch, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int* s_hist = s_dyn;               // [kBins] (16-byte aligned: read as int4)
  int* s_offs = s_hist + kBins;      // [B + 1] candidate offsets
  int* s_roots = s_offs + B + 1;     // [B] roots
  int* s_elig = s_roots + B;         // [B] eligible candidates e_b, then taken ones
  int* s_base = s_elig + B;          // [B] start of the request's sorted list
  int* s_noff = s_base + B;          // [B] packed offset of the request
  uint32_t* s_key = reinterpret_cast<uint32_t*>(s_noff + B);   // [num_candidates] sorted lists
  int* s_row = reinterpret_cast<int*>(s_key);                   // the same words: packed rows
  TL_TRACE_POINT(a, 8);

  // -- shape, roots, eligible counts --------------------------------------
  if (tid == 0) s_flag = 0;
  for (int b = tid; b <= B; b += kSelectThreads) s_offs[b] = a.cand_offsets[b];
  const int r_in = tid < B ? a.node_offsets[tid + 1] : 0;   // from launch 1
  for (int i = tid; i < kBins; i += kSelectThreads) s_hist[i] = 0;
  __syncthreads();
  int flags = 0, roots = 0, elig = 0;
  if (tid == 0) {
    flags |= s_offs[0] != 0;   // 1 = malformed offsets, 2 = a size or count out of range
    flags |= (s_offs[B] > a.num_candidates) << 1;
  }
  if (tid < B) {
    const int m = s_offs[tid + 1] - s_offs[tid];
    roots = r_in < 0 ? -r_in - 1 : r_in;
    flags |= m < 0;
    flags |= (m > kBudgetMaxTree || roots > a.max_nodes) << 1;
    // eligible: ranks below min(max_nodes - roots, non-roots); none if rejected
    elig = r_in < 0 ? 0 : max(0, min(a.max_nodes, m) - roots);
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
  // contiguous per-wave candidate segments, whole chunks of 64
  const int seg_len = (((M + kSelWaves - 1) / kSelWaves) + 63) & ~63;
  const int seg0 = wave * seg_len, seg1 = min(seg0 + seg_len, M);
  const int last = max(M - 1, 0);   // loads past the segment read this (in range) and are dropped
  // every rank of the segment, all loads in flight at once (kept for the packing)
  int r[kSegChunks];
  Cursor cur0 = {B - 1, M};
  if (M > 0) {
#pragma unroll
    for (int c = 0; c < kSegChunks; ++c) r[c] = a.rank[min(seg0 + 64 * c + lane, last)];
    cur0.seek(s_offs, B, min(seg0 + lane, last));
  }
  __syncthreads();   // s_base
  TL_TRACE_POINT(a, 9);

  int take = 0;   // this thread's request (tid < B): candidates taken
  if (K > 0 && K < E) {
    // -- eligible keys into per-request descending lists --------------------
    Cursor cu = cur0;
    int eb = s_elig[cu.b], bb = s_base[cu.b];
#pragma unroll
    for (int h = 0; h < kSegChunks; h += kSegChunks / 2) {   // half a segment of rho loads at a time
      float x[kSegChunks / 2];
#pragma unroll
      for (int c = 0; c < kSegChunks / 2; ++c) x[c] = a.rho[min(seg0 + 64 * (h + c) + lane, last)];
#pragma unroll
      for (int c = 0; c < kSegChunks / 2; ++c) {
        const int i = seg0 + 64 * (h + c) + lane;
        if (i < seg1) {
          if (cu.advance(s_offs, B, i)) {
            eb = s_elig[cu.b];
            bb = s_base[cu.b];
          }
          if (r[h + c] >= 0 && r[h + c] < eb) s_key[bb + r[h + c]] = __float_as_uint(x[c]) & 0x7fffffffu;
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
  __syncthreads();
  TL_TRACE_POINT(a, 12);

  // -- packing: the row of a selected node = selected candidates before it --
  // (roots have rank -1, a rejected request's other candidates never rank below its take)
  uint32_t selbits = 0;
  int count = 0;
  {
    Cursor cu = cur0;
    int tk = s_elig[cu.b];
#pragma unroll
    for (int c = 0; c < kSegChunks; ++c) {
      const int i = seg0 + 64 * c + lane;
      if (i < seg1) {
        if (cu.advance(s_offs, B, i)) tk = s_elig[cu.b];
        const bool sel = r[c] == -1 || (r[c] >= 0 && r[c] < tk);
        selbits |= (uint32_t)sel << c;
        count += sel;
      }
    }
  }
  const int wave_count = wave_sum(count);
  int all_sel;
  const int wave_incl = block_inclusive_scan<kSelWaves>(lane == 0 ? wave_count : 0, s_part, &all_sel);
  int row = __shfl(wave_incl, 0, 64) - wave_count;   // rows before this wave's segment
#pragma unroll
  for (int c = 0; c < kSegChunks; ++c) {
    const int i = seg0 + 64 * c + lane;
    const bool sel = (selbits >> c) & 1u;
    const uint64_t m = __ballot(sel);
    if (i < seg1) s_row[i] = sel ? row + lanes_below(m) : -1;
    row += __popcll(m);
  }
  TL_TRACE_POINT(a, 13);
  int p[kSegChunks];
  if (M > 0) {
#pragma unroll
    for (int c = 0; c < kSegChunks; ++c) {   // parents of the selected nodes only
      const int i = seg0 + 64 * c + lane;
      p[c] = a.cand_parent[((selbits >> c) & 1u) ? i : last];
    }
  }
  __syncthreads();
  TL_TRACE_POINT(a, 14);
  int broken = 0;
  {
    Cursor cu = cur0;
    int o0b = s_offs[cu.b], nb = s_noff[cu.b];
#pragma unroll
    for (int c = 0; c < kSegChunks; ++c) {
      if ((selbits >> c) & 1u) {
        const int i = seg0 + 64 * c + lane;
        if (cu.advance(s_offs, B, i)) {
          o0b = s_offs[cu.b];
          nb = s_noff[cu.b];
        }
        const int k = s_row[i];
        const int pp = p[c] == -1 ? -1 : s_row[o0b + p[c]] - nb;
        broken |= (p[c] != -1 && pp < 0) || k >= a.capacity;   // never for a consistent selection
        if (k < a.capacity) {
          a.src[k] = i;
          a.parent[k] = pp;
        }
      }
    }
  }
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
  hipLaunchKernelGGL(rho_rank_kernel, dim3((unsigned)a.batch), dim3(kRankThreads), 0, stream, a);
  hipLaunchKernelGGL(select_pack_kernel, dim3(1), dim3(kSelectThreads), lds, stream, a);
  return hipGetLastError() == hipSuccess ? TL_OK : TL_EHIP;
}

}  // namespace tl
