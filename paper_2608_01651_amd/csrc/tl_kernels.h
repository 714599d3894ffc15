// Internal interface between the C ABI (abi.cpp) and the kernel files.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "treelin.h"

namespace tl {

struct VerifyArgs {
  const int32_t* node_offsets;
  const int32_t* parent;
  const void* q;
  const void* k;
  const void* v;
  const float* g;
  const float* beta;
  const float* state;
  const int32_t* slot;
  float* out;
  int32_t* dev_err;
  int batch, Hk, Hv, max_nodes, num_slots;
  int tm;          // max_nodes rounded up to a multiple of 16
  int lds_bytes;   // dynamic LDS of the launch (set by the launcher)
  float q_scale;
#ifdef TL_TRACE
  long long* trace;  // [blocks][16] wall-clock stamps (trace builds only)
#endif
};

// What every commit launch shares: the forest, the slot map and the shape.
struct CommitCommon {
  const int32_t* node_offsets;
  const int32_t* parent;
  const int32_t* slot;
  int32_t* dev_err;
  int batch, Hk, Hv, max_nodes, num_slots;
#ifdef TL_TRACE
  long long* trace;  // [blocks][16] wall-clock stamps (trace builds only)
#endif
};

// One layer's per-node rows and state slots.
struct CommitLayer {
  const void* k;
  const void* v;
  const float* g;
  const float* beta;
  float* state;
};

// tree_state_commit: one layer, explicit root-first paths.
struct CommitArgs {
  CommitCommon c;
  CommitLayer ly;
  const int32_t* path_offsets;
  const int32_t* path;
};

// tree_state_commit_layers: up to kMaxCommitLayers layers in one launch, the
// accepted path of each request given by its terminal node.
// NL is the capacity of the layer table (the kernel argument's size): 1 for
// the launches that serve a single layer.
constexpr int kMaxCommitLayers = 64;
template <int NL>
struct CommitLayersArgsN {
  CommitCommon c;
  const int32_t* terminal;
  int num_layers;
  CommitLayer ly[NL];
};
using CommitLayersArgs = CommitLayersArgsN<kMaxCommitLayers>;

// tree_accepted_path
struct PathArgs {
  const int32_t* node_offsets;
  const int32_t* parent;
  const int32_t* terminal;
  int32_t* path_len;
  int32_t* path;
  int32_t* dev_err;
  int batch, max_nodes;
};

struct TopoArgs {
  const int32_t* node_offsets;
  const int32_t* parent;
  uint64_t* anc_mask;
  int32_t* depth;
  int32_t* dev_err;
  int batch, max_nodes, words;
};

// Channels per workgroup of the convolution-state commit (256 threads x 8);
// conv_gates picks its own channel tile by tree size.
constexpr int kConvCommitTile = 2048;

// tree_conv_gates
struct ConvArgs {
  const int32_t* node_offsets;
  const int32_t* parent;
  const void* x;
  const float* gate_a;
  const float* gate_b;
  const float* conv_weight;
  const float* conv_bias;
  const float* A_log;
  const float* dt_bias;
  const void* conv_state;
  const int32_t* slot;
  void* q;
  void* k;
  void* v;
  float* g;
  float* beta;
  int32_t* dev_err;
  int batch, Hk, Hv, dk, dv, C, max_nodes, num_slots;
  int tiles;   // channel tiles per request (set by the launcher)
  float eps;
#ifdef TL_TRACE
  long long* trace;  // [blocks][16] wall-clock stamps (trace builds only)
#endif
};

// tree_conv_state_commit
struct ConvCommitArgs {
  const int32_t* node_offsets;
  const int32_t* parent;
  const int32_t* terminal;
  const void* x;
  void* conv_state;
  const int32_t* slot;
  int32_t* dev_err;
  int batch, C, max_nodes, num_slots, tiles;
};

// tree_budget_select
constexpr int kBudgetMaxTree = 1024;          // candidates per request (one per thread)
constexpr int kBudgetMaxBatch = 1024;         // requests (one per selection thread)
constexpr int kBudgetMaxCandidates = 32768;   // candidates per batch (one workgroup's LDS)
constexpr int kSelectThreads = 1024;

// Bytes of the static workspace of tree_budget_select_noalloc (per GPU).
constexpr size_t kBudgetScratchBytes = TL_BUDGET_NOALLOC_MAX_BYTES;

// tree_budget_select's workspace, per request b (slots of max_nodes): its
// eligible candidates' rho bits in rank order, their request-local indices,
// its roots' indices, and {roots, eligible, rejected} counts.
struct BudgetWorkspace {
  size_t meta, key, cand, root, total;
};
inline BudgetWorkspace budget_workspace_layout(int batch, int max_nodes) {
  BudgetWorkspace w;
  size_t o = 0;
  w.meta = o; o += (size_t)batch * 16;
  w.key = o;  o += (size_t)batch * max_nodes * 4;
  w.cand = o; o += (size_t)batch * max_nodes * 4;
  w.root = o; o += ((size_t)batch * max_nodes * 2 + 15) / 16 * 16;
  w.total = (o + 255) / 256 * 256;
  return w;
}

struct BudgetArgs {
  const int32_t* cand_offsets;
  const int32_t* cand_parent;
  const float* cand_prob;
  float* rho;
  int32_t* rank;
  int32_t* node_offsets;
  int32_t* parent;
  int32_t* src;
  int32_t* dev_err;
  int32_t* ws_meta;    // [batch][4]
  uint32_t* ws_key;    // [batch][max_nodes]
  uint32_t* ws_cand;   // [batch][max_nodes]: index | (parent + 1) << 16
  uint16_t* ws_root;   // [batch][max_nodes]
  int batch, max_nodes, num_candidates, capacity;
#ifdef TL_TRACE
  long long* trace;  // [blocks][16] wall-clock stamps (trace builds only)
#endif
};

tl_status launch_verify(const tl_problem& p, const VerifyArgs& a, hipStream_t stream);
tl_status launch_verify_tiled(const tl_problem& p, const VerifyArgs& a, hipStream_t stream);
tl_status launch_verify_gdn_dense(const tl_problem& p, const VerifyArgs& a, hipStream_t stream);
tl_status launch_verify_gla_large(const tl_problem& p, const VerifyArgs& a, hipStream_t stream);
int verify_gla_large_lds_bytes(int d, int tm);
int verify_tiled_lds_bytes(int d, int tm, int W);
tl_status launch_commit(const tl_problem& p, const CommitArgs& a, hipStream_t stream);
tl_status launch_commit_layers(const tl_problem& p, const CommitLayersArgs& a, hipStream_t stream);
tl_status launch_accepted_path(const PathArgs& a, hipStream_t stream);
tl_status launch_topology(const tl_problem& p, const TopoArgs& a, hipStream_t stream);
tl_status launch_conv_gates(const ConvArgs& a, int width, bool gdn, hipStream_t stream);
tl_status launch_conv_state_commit(const ConvCommitArgs& a, int width, hipStream_t stream);
tl_status launch_budget_select(const BudgetArgs& a, hipStream_t stream);
// Device address of the current device's static budget workspace (the
// kBudgetScratchBytes array of tree_budget_select_noalloc).
tl_status budget_scratch(void** ptr);
int budget_select_lds_bytes(int batch, int num_candidates);
int verify_lds_bytes(const tl_problem& p, int tm);

}  // namespace tl
