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
  float q_scale;
#ifdef TL_TRACE
  long long* trace;  // [blocks][16] wall-clock stamps (trace builds only)
#endif
};

struct CommitArgs {
  const int32_t* node_offsets;
  const int32_t* parent;
  const int32_t* path_offsets;
  const int32_t* path;
  const void* k;
  const void* v;
  const float* g;
  const float* beta;
  float* state;
  const int32_t* slot;
  int32_t* dev_err;
  int batch, Hk, Hv, max_nodes, num_slots;
#ifdef TL_TRACE
  long long* trace;  // [blocks][16] wall-clock stamps (trace builds only)
#endif
};

struct TopoArgs {
  const int32_t* node_offsets;
  const int32_t* parent;
  uint64_t* anc_mask;
  int32_t* depth;
  int32_t* dev_err;
  int batch, max_nodes, words;
};

tl_status launch_verify(const tl_problem& p, const VerifyArgs& a, hipStream_t stream);
tl_status launch_verify_tiled(const tl_problem& p, const VerifyArgs& a, hipStream_t stream);
int verify_tiled_lds_bytes(int mode, int d, int tm, int W);
tl_status launch_commit(const tl_problem& p, const CommitArgs& a, hipStream_t stream);
tl_status launch_topology(const TopoArgs& a, hipStream_t stream);
int verify_lds_bytes(const tl_problem& p, int tm);

}  // namespace tl
