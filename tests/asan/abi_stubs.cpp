// Host-only stand-ins for the kernel launchers behind the C ABI, for the
// sanitizer build of abi.cpp: each records what the ABI handed it (so the
// driver can check the argument marshalling) and launches nothing.
#include "abi_stubs.h"

namespace stub {
Calls calls;
}

namespace tl {

tl_status launch_verify(const tl_problem& p, const VerifyArgs& a, hipStream_t) {
  stub::calls.verify++;
  stub::calls.problem = p;
  stub::calls.verify_args = a;
  return TL_OK;
}
tl_status launch_verify_tiled(const tl_problem&, const VerifyArgs&, hipStream_t) { return TL_OK; }
int verify_tiled_lds_bytes(int, int, int, int) { return 0; }
tl_status launch_commit(const tl_problem& p, const CommitArgs& a, hipStream_t) {
  stub::calls.commit++;
  stub::calls.problem = p;
  stub::calls.commit_args = a;
  return TL_OK;
}
tl_status launch_commit_layers(const tl_problem&, const CommitLayersArgs& a, hipStream_t) {
  stub::calls.commit_layers++;
  stub::calls.num_layers = a.num_layers;
  stub::calls.last_layer_state = a.num_layers > 0 ? a.ly[a.num_layers - 1].state : nullptr;
  stub::calls.unused_layer_state = a.num_layers < kMaxCommitLayers ? a.ly[a.num_layers].state : nullptr;
  return TL_OK;
}
tl_status launch_accepted_path(const PathArgs&, hipStream_t) {
  stub::calls.path++;
  return TL_OK;
}
tl_status launch_topology(const tl_problem&, const TopoArgs& a, hipStream_t) {
  stub::calls.topology++;
  stub::calls.topo_words = a.words;
  return TL_OK;
}
tl_status launch_conv_gates(const ConvArgs& a, int width, bool gdn, hipStream_t) {
  stub::calls.conv++;
  stub::calls.conv_channels = a.C;
  stub::calls.conv_width = width;
  stub::calls.conv_gdn = gdn;
  return TL_OK;
}
tl_status launch_conv_state_commit(const ConvCommitArgs& a, int, hipStream_t) {
  stub::calls.conv_commit++;
  stub::calls.conv_commit_tiles = a.tiles;
  return TL_OK;
}
tl_status launch_budget_select(const BudgetArgs& a, hipStream_t) {
  stub::calls.budget++;
  stub::calls.budget_args = a;
  return TL_OK;
}
tl_status budget_scratch(void** ptr) {
  stub::calls.scratch++;
  *ptr = stub::calls.scratch_base;
  return TL_OK;
}

}  // namespace tl
