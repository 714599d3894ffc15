// Shared pieces of the verify kernel: LDS layout of the vector and delta-rule
// paths, the unit of work, and the dynamic LDS array.
#pragma once

#include <hip/hip_runtime.h>

#include "tl_device.h"
#include "tl_kernels.h"

namespace tl {

extern __shared__ __align__(16) unsigned char tl_lds[];

// Debug builds (-DTL_DEBUG): every word of the launch's dynamic LDS is
// filled with NaN (0xFFC0 in each bf16 half) before any other access, so
// that a read of LDS the kernel has not written shows up in its results.
// Called by every thread, before any early return.  Empty otherwise.
__device__ inline void lds_poison(int bytes) {
#ifdef TL_DEBUG
  for (int x = (int)threadIdx.x * 4; x < bytes; x += (int)blockDim.x * 4)
    *reinterpret_cast<uint32_t*>(tl_lds + x) = 0xFFC0FFC0u;
  __syncthreads();
#else
  (void)bytes;
#endif
}

// ---------------------------------------------------------------------------
// LDS layout (bytes); identical on host and device.
// ---------------------------------------------------------------------------
struct VerifyLayout {
  int par, depth, cl, beta, mask, tmask, qst, kst, vst, ubuf, uni, total;
};

__host__ __device__ inline int align16(int x) { return (x + 15) & ~15; }

__host__ __device__ inline VerifyLayout verify_layout(int mode, int D, int BV, int vbytes, int tm,
                                                      int W, bool mfma) {
  const bool gdn = (mode == TL_MODE_GDN);
  VerifyLayout L;
  int o = 0;
  L.par = o;   o += align16(tm * 4);
  L.depth = o; o += align16(tm * 4);
  L.cl = o;    o += align16(tm * 4);
  L.beta = o;  o += gdn ? align16(tm * 4) : 0;
  L.mask = o;  o += tm * W * 8;
  L.tmask = o; o += align16((tm / kTile) * W * 8);
  L.qst = o;   o += (mfma && W == 1) ? tm * D * 2 : 0;     // Q rows (trees of <= 64 nodes)
  L.kst = o;   o += mfma ? tm * D * 2 : 0;                 // K rows, swizzled bf16
  L.vst = o;   o += gdn ? 0 : tm * BV * vbytes;            // value slice (GLA)
  L.ubuf = o;  o += gdn ? tm * BV * 4 : 0;                 // U rows (delta rule)
  L.uni = o;
  // union: topology scratch | per-tile coefficients (c, and G for the delta rule)
  const int topo = kThreads * (4 + 4 + 4) + kThreads * W * 8;
  const int ng = mfma ? 4 / W : 1;   // node tiles whose coefficients are kept at once
  const int coef = ng * kTile * tm * 4 * (gdn ? 2 : 1);
  o += align16(topo > coef ? topo : coef);
  L.total = o;
  return L;
}

struct Unit {
  int b, h, hq, slice, off, T, sidx, tm;
};

// C operand fragments of a tree of nt node tiles (trees of <= 64 nodes): tile
// I uses I / 2 + 1 chunks of 32 ancestor columns.
__host__ __device__ constexpr int gla_small_slots(int nt) { return (nt * nt + 2 * nt + (nt & 1)) / 4; }

}  // namespace tl
