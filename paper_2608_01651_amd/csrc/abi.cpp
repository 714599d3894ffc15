// C ABI of libtreelin: synchronous argument checks, then one launch on the
// caller's stream.  Nothing is allocated and no state is kept between calls.
#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "tl_kernels.h"
#include "treelin.h"

namespace {

#ifdef TL_TRACE
long long* g_trace = nullptr;
#endif

bool aligned(const void* p, uintptr_t n) { return (reinterpret_cast<uintptr_t>(p) % n) == 0; }

bool supported_d(int d) { return d == 16 || d == 32 || d == 64 || d == 128; }

// Checks shared by every entry point.  Returns TL_OK or the failing status.
tl_status check_problem(const tl_problem* p) {
  if (!p) return TL_EINVAL;
  if (p->batch < 0 || p->num_qk_heads < 1 || p->num_v_heads < 1) return TL_EINVAL;
  if (p->num_v_heads % p->num_qk_heads) return TL_EINVAL;
  if (p->mode != TL_MODE_GLA && p->mode != TL_MODE_GDN) return TL_EINVAL;
  if (p->in_dtype != TL_BF16 && p->in_dtype != TL_F32) return TL_EINVAL;
  if (!supported_d(p->d_k) || p->d_v != p->d_k) return TL_EUNSUPPORTED;
  if (p->max_nodes < 1 || p->max_nodes > 256) return TL_EUNSUPPORTED;
  if (p->batch > 0) {
    if (p->num_slots < 1) return TL_EINVAL;
    const long units = (long)p->batch * p->num_v_heads;
    if (units > (1L << 30)) return TL_EINVAL;
  }
  return TL_OK;
}

tl_status check_tensors(const tl_problem* p, const int32_t* node_offsets, const int32_t* parent,
                        const void* k, const void* v, const float* g, const float* beta,
                        const void* state, const int32_t* slot) {
  if (!node_offsets || !parent || !k || !v || !g || !state) return TL_EINVAL;
  if ((p->mode == TL_MODE_GLA) != (beta == nullptr)) return TL_EINVAL;
  if (!aligned(node_offsets, 4) || !aligned(parent, 4) || !aligned(g, 4)) return TL_EINVAL;
  if (beta && !aligned(beta, 4)) return TL_EINVAL;
  if (slot && !aligned(slot, 4)) return TL_EINVAL;
  if (!aligned(k, 16) || !aligned(v, 16) || !aligned(state, 16)) return TL_EINVAL;
  if (!slot && p->num_slots < p->batch) return TL_EINVAL;
  return TL_OK;
}

void fill_common(const tl_problem* p, const int32_t* node_offsets, const int32_t* parent,
                 const int32_t* slot, int32_t* dev_err, tl::CommitCommon& c) {
  c.node_offsets = node_offsets;
  c.parent = parent;
  c.slot = slot;
  c.dev_err = dev_err;
  c.batch = p->batch;
  c.Hk = p->num_qk_heads;
  c.Hv = p->num_v_heads;
  c.max_nodes = p->max_nodes;
  c.num_slots = p->num_slots;
#ifdef TL_TRACE
  c.trace = g_trace;
#endif
}

}  // namespace

extern "C" {

#ifdef TL_TRACE
// Trace builds only: stamps of the next verify launches go to p ([blocks][16]).
void tl_set_trace(long long* p) { g_trace = p; }
#endif

size_t tl_workspace_bytes(const tl_problem* problem) {
  // every intermediate of verification (masks, decays, C, G, U, B0) lives in
  // registers and LDS: no layer-local device scratch
  (void)problem;
  return 0;
}

tl_status tree_lin_attn_verify(const tl_problem* problem, const int32_t* node_offsets,
                               const int32_t* parent, const void* q, const void* k, const void* v,
                               const float* g, const float* beta, const float* state,
                               const int32_t* slot, float* out, int32_t* dev_err,
                               void* workspace, size_t workspace_bytes, void* stream) {
  tl_status st = check_problem(problem);
  if (st != TL_OK) return st;
  if (workspace_bytes < tl_workspace_bytes(problem)) return TL_EINVAL;
  if (workspace_bytes > 0 && (!workspace || !aligned(workspace, 256))) return TL_EINVAL;
  if (problem->batch == 0) return TL_OK;
  st = check_tensors(problem, node_offsets, parent, k, v, g, beta, state, slot);
  if (st != TL_OK) return st;
  if (!q || !out || !aligned(q, 16) || !aligned(out, 16)) return TL_EINVAL;
  if (dev_err && !aligned(dev_err, 4)) return TL_EINVAL;
  tl::VerifyArgs a;
  a.node_offsets = node_offsets;
  a.parent = parent;
  a.q = q;
  a.k = k;
  a.v = v;
  a.g = g;
  a.beta = beta;
  a.state = state;
  a.slot = slot;
  a.out = out;
  a.dev_err = dev_err;
  a.batch = problem->batch;
  a.Hk = problem->num_qk_heads;
  a.Hv = problem->num_v_heads;
  a.max_nodes = problem->max_nodes;
  a.num_slots = problem->num_slots;
  a.tm = (problem->max_nodes + 15) & ~15;
  a.lds_bytes = 0;
  a.q_scale = problem->q_scale;
#ifdef TL_TRACE
  a.trace = g_trace;
#endif
  return tl::launch_verify(*problem, a, reinterpret_cast<hipStream_t>(stream));
}

tl_status tree_state_commit(const tl_problem* problem, const int32_t* node_offsets,
                            const int32_t* parent, const int32_t* path_offsets, const int32_t* path,
                            const void* k, const void* v, const float* g, const float* beta,
                            float* state, const int32_t* slot, int32_t* dev_err, void* stream) {
  tl_status st = check_problem(problem);
  if (st != TL_OK) return st;
  if (problem->batch == 0) return TL_OK;
  st = check_tensors(problem, node_offsets, parent, k, v, g, beta, state, slot);
  if (st != TL_OK) return st;
  if (!path_offsets || !aligned(path_offsets, 4)) return TL_EINVAL;
  if (path && !aligned(path, 4)) return TL_EINVAL;
  if (dev_err && !aligned(dev_err, 4)) return TL_EINVAL;
  tl::CommitArgs a;
  fill_common(problem, node_offsets, parent, slot, dev_err, a.c);
  a.ly = tl::CommitLayer{k, v, g, beta, state};
  a.path_offsets = path_offsets;
  a.path = path;   // NULL is allowed when every path is empty
  return tl::launch_commit(*problem, a, reinterpret_cast<hipStream_t>(stream));
}

tl_status tree_state_commit_layers(const tl_problem* problem, int32_t num_layers,
                                   const tl_layer* layers, const int32_t* node_offsets,
                                   const int32_t* parent, const int32_t* terminal,
                                   const int32_t* slot, int32_t* dev_err, void* stream) {
  tl_status st = check_problem(problem);
  if (st != TL_OK) return st;
  if (num_layers < 0 || num_layers > TL_MAX_COMMIT_LAYERS) return TL_EINVAL;
  if (problem->batch == 0 || num_layers == 0) return TL_OK;
  if (!layers || !terminal || !aligned(terminal, 4)) return TL_EINVAL;
  if (dev_err && !aligned(dev_err, 4)) return TL_EINVAL;
  tl::CommitLayersArgs a;
  fill_common(problem, node_offsets, parent, slot, dev_err, a.c);
  a.terminal = terminal;
  a.num_layers = num_layers;
  for (int l = 0; l < num_layers; ++l) {
    const tl_layer& L = layers[l];
    st = check_tensors(problem, node_offsets, parent, L.k, L.v, L.g, L.beta, L.state, slot);
    if (st != TL_OK) return st;
    a.ly[l] = tl::CommitLayer{L.k, L.v, L.g, L.beta, L.state};
  }
  for (int l = num_layers; l < tl::kMaxCommitLayers; ++l) a.ly[l] = tl::CommitLayer{};
  return tl::launch_commit_layers(*problem, a, reinterpret_cast<hipStream_t>(stream));
}

tl_status tree_accepted_path(const tl_problem* problem, const int32_t* node_offsets,
                             const int32_t* parent, const int32_t* terminal, int32_t* path_len,
                             int32_t* path, int32_t* dev_err, void* stream) {
  tl_status st = check_problem(problem);
  if (st != TL_OK) return st;
  if (problem->batch == 0) return TL_OK;
  if (!node_offsets || !parent || !terminal || !path_len || !path) return TL_EINVAL;
  if (!aligned(node_offsets, 4) || !aligned(parent, 4) || !aligned(terminal, 4) ||
      !aligned(path_len, 4) || !aligned(path, 4))
    return TL_EINVAL;
  if (dev_err && !aligned(dev_err, 4)) return TL_EINVAL;
  tl::PathArgs a;
  a.node_offsets = node_offsets;
  a.parent = parent;
  a.terminal = terminal;
  a.path_len = path_len;
  a.path = path;
  a.dev_err = dev_err;
  a.batch = problem->batch;
  a.max_nodes = problem->max_nodes;
  return tl::launch_accepted_path(a, reinterpret_cast<hipStream_t>(stream));
}

tl_status tree_topology_export(const tl_problem* problem, const int32_t* node_offsets,
                               const int32_t* parent, uint64_t* anc_mask, int32_t* depth,
                               int32_t* dev_err, void* stream) {
  tl_status st = check_problem(problem);
  if (st != TL_OK) return st;
  if (problem->batch == 0) return TL_OK;
  if (!node_offsets || !parent || !anc_mask || !depth) return TL_EINVAL;
  if (!aligned(node_offsets, 4) || !aligned(parent, 4) || !aligned(anc_mask, 8) ||
      !aligned(depth, 4))
    return TL_EINVAL;
  if (dev_err && !aligned(dev_err, 4)) return TL_EINVAL;
  tl::TopoArgs a;
  a.node_offsets = node_offsets;
  a.parent = parent;
  a.anc_mask = anc_mask;
  a.depth = depth;
  a.dev_err = dev_err;
  a.batch = problem->batch;
  a.max_nodes = problem->max_nodes;
  a.words = (problem->max_nodes + 63) / 64;
  return tl::launch_topology(*problem, a, reinterpret_cast<hipStream_t>(stream));
}

tl_status tree_conv_gates(const tl_problem* problem, int32_t conv_width, float norm_eps,
                          const int32_t* node_offsets, const int32_t* parent, const void* x,
                          const float* gate_a, const float* gate_b, const float* conv_weight,
                          const float* conv_bias, const float* A_log, const float* dt_bias,
                          const void* conv_state, const int32_t* slot, void* q, void* k, void* v,
                          float* g, float* beta, int32_t* dev_err, void* stream) {
  tl_status st = check_problem(problem);
  if (st != TL_OK) return st;
  if (conv_width < 2 || conv_width > 4 || problem->in_dtype != TL_BF16) return TL_EUNSUPPORTED;
  if (!(norm_eps >= 0.f)) return TL_EINVAL;
  if (problem->batch == 0) return TL_OK;
  const bool gdn = problem->mode == TL_MODE_GDN;
  if (!node_offsets || !parent || !x || !gate_a || !conv_weight || !conv_bias || !A_log ||
      !dt_bias || !conv_state || !q || !k || !v || !g)
    return TL_EINVAL;
  if (gdn != (gate_b != nullptr) || gdn != (beta != nullptr)) return TL_EINVAL;
  if (!aligned(x, 16) || !aligned(conv_state, 16) || !aligned(q, 16) || !aligned(k, 16) ||
      !aligned(v, 16) || !aligned(conv_weight, 16) || !aligned(conv_bias, 16))
    return TL_EINVAL;
  if (!aligned(node_offsets, 4) || !aligned(parent, 4) || !aligned(gate_a, 4) || !aligned(A_log, 4) ||
      !aligned(dt_bias, 4) || !aligned(g, 4) || (gate_b && !aligned(gate_b, 4)) ||
      (beta && !aligned(beta, 4)) || (slot && !aligned(slot, 4)) || (dev_err && !aligned(dev_err, 4)))
    return TL_EINVAL;
  if (!slot && problem->num_slots < problem->batch) return TL_EINVAL;
  tl::ConvArgs a;
  a.node_offsets = node_offsets;
  a.parent = parent;
  a.x = x;
  a.gate_a = gate_a;
  a.gate_b = gate_b;
  a.conv_weight = conv_weight;
  a.conv_bias = conv_bias;
  a.A_log = A_log;
  a.dt_bias = dt_bias;
  a.conv_state = conv_state;
  a.slot = slot;
  a.q = q;
  a.k = k;
  a.v = v;
  a.g = g;
  a.beta = beta;
  a.dev_err = dev_err;
  a.batch = problem->batch;
  a.Hk = problem->num_qk_heads;
  a.Hv = problem->num_v_heads;
  a.dk = problem->d_k;
  a.dv = problem->d_v;
  a.C = 2 * a.Hk * a.dk + a.Hv * a.dv;
  a.max_nodes = problem->max_nodes;
  a.num_slots = problem->num_slots;
  a.tiles = 0;
  a.eps = norm_eps;
#ifdef TL_TRACE
  a.trace = g_trace;
#endif
  return tl::launch_conv_gates(a, conv_width, gdn, reinterpret_cast<hipStream_t>(stream));
}

tl_status tree_conv_state_commit(const tl_problem* problem, int32_t conv_width,
                                 const int32_t* node_offsets, const int32_t* parent,
                                 const int32_t* terminal, const void* x, void* conv_state,
                                 const int32_t* slot, int32_t* dev_err, void* stream) {
  tl_status st = check_problem(problem);
  if (st != TL_OK) return st;
  if (conv_width < 2 || conv_width > 4 || problem->in_dtype != TL_BF16) return TL_EUNSUPPORTED;
  if (problem->batch == 0) return TL_OK;
  if (!node_offsets || !parent || !terminal || !x || !conv_state) return TL_EINVAL;
  if (!aligned(x, 16) || !aligned(conv_state, 16) || !aligned(node_offsets, 4) ||
      !aligned(parent, 4) || !aligned(terminal, 4) || (slot && !aligned(slot, 4)) ||
      (dev_err && !aligned(dev_err, 4)))
    return TL_EINVAL;
  if (!slot && problem->num_slots < problem->batch) return TL_EINVAL;
  tl::ConvCommitArgs a;
  a.node_offsets = node_offsets;
  a.parent = parent;
  a.terminal = terminal;
  a.x = x;
  a.conv_state = conv_state;
  a.slot = slot;
  a.dev_err = dev_err;
  a.batch = problem->batch;
  a.C = 2 * problem->num_qk_heads * problem->d_k + problem->num_v_heads * problem->d_v;
  a.max_nodes = problem->max_nodes;
  a.num_slots = problem->num_slots;
  a.tiles = (a.C + tl::kConvCommitTile - 1) / tl::kConvCommitTile;
  return tl::launch_conv_state_commit(a, conv_width, reinterpret_cast<hipStream_t>(stream));
}

size_t tree_budget_workspace_bytes(int32_t batch, int32_t max_nodes) {
  if (batch <= 0 || max_nodes <= 0) return 0;
  return tl::budget_workspace_layout(batch, max_nodes).total;
}

}  // extern "C"

namespace {

// Host checks of both budget entry points; on TL_OK `W` is the workspace
// layout the problem needs.
tl_status check_budget(const tl_problem* problem, int32_t num_candidates, int32_t capacity,
                       const int32_t* cand_offsets, const int32_t* cand_parent,
                       const float* cand_prob, const float* rho, const int32_t* rank,
                       const int32_t* node_offsets, const int32_t* parent, const int32_t* src,
                       const int32_t* dev_err, tl::BudgetWorkspace& W) {
  tl_status st = check_problem(problem);
  if (st != TL_OK) return st;
  if (problem->batch == 0) return TL_OK;
  if (num_candidates < 0 || capacity < 0) return TL_EINVAL;
  if (problem->batch > tl::kBudgetMaxBatch || num_candidates > tl::kBudgetMaxCandidates)
    return TL_EUNSUPPORTED;
  if (!cand_offsets || !cand_parent || !cand_prob || !rho || !rank || !node_offsets || !parent ||
      !src)
    return TL_EINVAL;
  if (!aligned(cand_offsets, 4) || !aligned(cand_parent, 4) || !aligned(cand_prob, 4) ||
      !aligned(rho, 4) || !aligned(rank, 4) || !aligned(node_offsets, 4) || !aligned(parent, 4) ||
      !aligned(src, 4))
    return TL_EINVAL;
  if (dev_err && !aligned(dev_err, 4)) return TL_EINVAL;
  W = tl::budget_workspace_layout(problem->batch, problem->max_nodes);
  return TL_OK;
}

tl_status launch_budget(const tl_problem* problem, int32_t num_candidates, int32_t capacity,
                        const int32_t* cand_offsets, const int32_t* cand_parent,
                        const float* cand_prob, float* rho, int32_t* rank, int32_t* node_offsets,
                        int32_t* parent, int32_t* src, const tl::BudgetWorkspace& W, void* workspace,
                        int32_t* dev_err, void* stream) {
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  tl::BudgetArgs a;
  a.cand_offsets = cand_offsets;
  a.cand_parent = cand_parent;
  a.cand_prob = cand_prob;
  a.rho = rho;
  a.rank = rank;
  a.node_offsets = node_offsets;
  a.parent = parent;
  a.src = src;
  a.dev_err = dev_err;
  a.ws_meta = reinterpret_cast<int32_t*>(ws + W.meta);
  a.ws_key = reinterpret_cast<uint32_t*>(ws + W.key);
  a.ws_cand = reinterpret_cast<uint32_t*>(ws + W.cand);
  a.ws_root = reinterpret_cast<uint16_t*>(ws + W.root);
  a.batch = problem->batch;
  a.max_nodes = problem->max_nodes;
  a.num_candidates = num_candidates;
  a.capacity = capacity;
#ifdef TL_TRACE
  a.trace = g_trace;
#endif
  return tl::launch_budget_select(a, reinterpret_cast<hipStream_t>(stream));
}

}  // namespace

extern "C" {

tl_status tree_budget_select(const tl_problem* problem, int32_t num_candidates, int32_t capacity,
                             const int32_t* cand_offsets, const int32_t* cand_parent,
                             const float* cand_prob, float* rho, int32_t* rank,
                             int32_t* node_offsets, int32_t* parent, int32_t* src,
                             void* workspace, size_t workspace_bytes,
                             int32_t* dev_err, void* stream) {
  tl::BudgetWorkspace W{};
  tl_status st = check_budget(problem, num_candidates, capacity, cand_offsets, cand_parent,
                              cand_prob, rho, rank, node_offsets, parent, src, dev_err, W);
  if (st != TL_OK || problem->batch == 0) return st;
  if (!workspace || !aligned(workspace, 256)) return TL_EINVAL;
  if (workspace_bytes < W.total) return TL_EINVAL;
  return launch_budget(problem, num_candidates, capacity, cand_offsets, cand_parent, cand_prob, rho,
                       rank, node_offsets, parent, src, W, workspace, dev_err, stream);
}

tl_status tree_budget_select_noalloc(const tl_problem* problem, int32_t num_candidates,
                                     int32_t capacity, const int32_t* cand_offsets,
                                     const int32_t* cand_parent, const float* cand_prob,
                                     float* rho, int32_t* rank, int32_t* node_offsets,
                                     int32_t* parent, int32_t* src, int32_t* dev_err,
                                     void* stream) {
  tl::BudgetWorkspace W{};
  tl_status st = check_budget(problem, num_candidates, capacity, cand_offsets, cand_parent,
                              cand_prob, rho, rank, node_offsets, parent, src, dev_err, W);
  if (st != TL_OK || problem->batch == 0) return st;
  if (W.total > tl::kBudgetScratchBytes) return TL_EUNSUPPORTED;   // beyond the static buffer
  void* ws = nullptr;
  st = tl::budget_scratch(&ws);
  if (st != TL_OK) return st;
  return launch_budget(problem, num_candidates, capacity, cand_offsets, cand_parent, cand_prob, rho,
                       rank, node_offsets, parent, src, W, ws, dev_err, stream);
}

const char* tl_status_string(tl_status s) {
  switch (s) {
    case TL_OK: return "TL_OK: success";
    case TL_EINVAL: return "TL_EINVAL: invalid argument";
    case TL_EBADTREE: return "TL_EBADTREE: malformed forest (offsets or parent array)";
    case TL_EBADPATH: return "TL_EBADPATH: accepted path is not a root-first chain";
    case TL_EUNSUPPORTED: return "TL_EUNSUPPORTED: unsupported head dimension or max_nodes";
    case TL_EHIP: return "TL_EHIP: HIP runtime error";
  }
  return "unknown tl_status";
}

const char* tl_version(void) { return "0.1.0"; }

}  // extern "C"
