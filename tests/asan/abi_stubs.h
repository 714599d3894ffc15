// What the launcher stand-ins record (sanitizer build of the C ABI).
#pragma once

#include "tl_kernels.h"

namespace stub {
struct Calls {
  int verify = 0, commit = 0, commit_layers = 0, path = 0, topology = 0, conv = 0,
      conv_commit = 0, budget = 0, scratch = 0;
  tl_problem problem{};
  tl::VerifyArgs verify_args{};
  tl::CommitArgs commit_args{};
  int num_layers = -1;
  float* last_layer_state = nullptr;
  float* unused_layer_state = nullptr;
  int topo_words = -1;
  int conv_channels = -1, conv_width = -1;
  bool conv_gdn = false;
  int conv_commit_tiles = -1;
  tl::BudgetArgs budget_args{};
  void* scratch_base = nullptr;
};
extern Calls calls;
}  // namespace stub
