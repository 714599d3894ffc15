// Drives every entry point of the C ABI (abi.cpp built for the host with
// AddressSanitizer and UndefinedBehaviorSanitizer, launchers replaced by the
// recording stand-ins of abi_stubs.cpp): the synchronous checks return the
// documented codes, valid calls reach the launcher with the fields the
// kernels rely on, and nothing reads or writes outside what it was given
// (the layer table, the problem struct).  Device pointers are fake aligned
// addresses that nothing dereferences.  Exit status 0 = every check held.
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "abi_stubs.h"
#include "treelin.h"

static int failures = 0;
#define CHECK(cond)                                                     \
  do {                                                                  \
    if (!(cond)) {                                                      \
      std::fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                       \
    }                                                                   \
  } while (0)

static void* P(uintptr_t a) { return reinterpret_cast<void*>(a); }
template <class T>
static T* F(uintptr_t a) { return reinterpret_cast<T*>(a); }

static tl_problem problem(int batch, int hk, int hv, int d, int max_nodes, int mode) {
  tl_problem p;
  std::memset(&p, 0, sizeof p);
  p.batch = batch;
  p.num_qk_heads = hk;
  p.num_v_heads = hv;
  p.d_k = p.d_v = d;
  p.max_nodes = max_nodes;
  p.num_slots = batch;
  p.mode = mode;
  p.in_dtype = TL_BF16;
  p.q_scale = 0.5f;
  return p;
}

static tl_status verify(const tl_problem* p, const float* beta = nullptr, void* ws = nullptr,
                        size_t ws_bytes = 0, void* q = P(0x10000)) {
  return tree_lin_attn_verify(p, F<const int32_t>(0x1000), F<const int32_t>(0x2000), q, P(0x20000),
                              P(0x30000), F<const float>(0x3000), beta, F<const float>(0x40000), nullptr,
                              F<float>(0x50000), F<int32_t>(0x4000), ws, ws_bytes, nullptr);
}

int main() {
  // ---- status strings
  for (int s = 0; s <= 5; ++s) CHECK(std::strncmp(tl_status_string((tl_status)s), "TL_", 3) == 0);
  CHECK(std::strstr(tl_status_string((tl_status)42), "unknown") != nullptr);
  CHECK(std::strlen(tl_version()) >= 5);

  // ---- verify
  tl_problem p = problem(32, 16, 32, 128, 64, TL_MODE_GLA);
  CHECK(verify(nullptr) == TL_EINVAL);
  CHECK(verify(&p) == TL_OK);
  CHECK(stub::calls.verify == 1);
  CHECK(stub::calls.verify_args.tm == 64 && stub::calls.verify_args.batch == 32);
  CHECK(stub::calls.verify_args.Hk == 16 && stub::calls.verify_args.Hv == 32);
  CHECK(stub::calls.verify_args.q_scale == 0.5f && stub::calls.verify_args.lds_bytes == 0);
  CHECK(stub::calls.verify_args.beta == nullptr && stub::calls.verify_args.slot == nullptr);
  tl_problem p2 = problem(3, 2, 4, 64, 130, TL_MODE_GDN);
  CHECK(verify(&p2) == TL_EINVAL);                        // the delta rule needs beta
  CHECK(verify(&p2, F<const float>(0x6000)) == TL_OK);
  CHECK(stub::calls.verify_args.tm == 144);
  CHECK(verify(&p, nullptr, nullptr, 0, P(0x10008)) == TL_EINVAL);   // q misaligned
  // the layer-local workspace: size 0 for every problem; a buffer that is passed is checked
  CHECK(tl_workspace_bytes(&p) == 0 && tl_workspace_bytes(&p2) == 0 && tl_workspace_bytes(nullptr) == 0);
  CHECK(verify(&p, nullptr, nullptr, 256) == TL_EINVAL);
  CHECK(verify(&p, nullptr, P(0x70010), 256) == TL_EINVAL);
  CHECK(verify(&p, nullptr, P(0x70000), 256) == TL_OK);
  tl_problem bad = p;
  bad.num_v_heads = 24;                                   // Hv % Hk != 0
  CHECK(verify(&bad) == TL_EINVAL);
  bad = p;
  bad.max_nodes = 257;
  CHECK(verify(&bad) == TL_EUNSUPPORTED);
  bad = p;
  bad.d_v = 64;
  CHECK(verify(&bad) == TL_EUNSUPPORTED);
  const int before = stub::calls.verify;
  tl_problem empty = problem(0, 1, 1, 32, 16, TL_MODE_GLA);
  CHECK(tree_lin_attn_verify(&empty, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                             nullptr, nullptr, nullptr, nullptr, nullptr, 0, nullptr) == TL_OK);
  CHECK(stub::calls.verify == before);                    // nothing launched

  // ---- commit
  CHECK(tree_state_commit(&p, F<const int32_t>(0x1000), F<const int32_t>(0x2000), F<const int32_t>(0x5000),
                          nullptr, P(0x20000), P(0x30000), F<const float>(0x3000), nullptr,
                          F<float>(0x40000), nullptr, nullptr, nullptr) == TL_OK);
  CHECK(stub::calls.commit == 1 && stub::calls.commit_args.path == nullptr);
  CHECK(stub::calls.commit_args.c.max_nodes == 64 && stub::calls.commit_args.c.num_slots == 32);
  CHECK(tree_state_commit(&p, F<const int32_t>(0x1000), F<const int32_t>(0x2000), nullptr, nullptr,
                          P(0x20000), P(0x30000), F<const float>(0x3000), nullptr, F<float>(0x40000),
                          nullptr, nullptr, nullptr) == TL_EINVAL);

  // ---- unified commit: the layer table is read exactly num_layers entries deep
  std::vector<tl_layer> layers(TL_MAX_COMMIT_LAYERS);
  for (int l = 0; l < TL_MAX_COMMIT_LAYERS; ++l)
    layers[l] = tl_layer{P(0x20000), P(0x30000), F<const float>(0x3000), nullptr,
                         F<float>(0x100000 + 0x10000 * (uintptr_t)l)};
  CHECK(tree_state_commit_layers(&p, TL_MAX_COMMIT_LAYERS, layers.data(), F<const int32_t>(0x1000),
                                 F<const int32_t>(0x2000), F<const int32_t>(0x5000), nullptr, nullptr,
                                 nullptr) == TL_OK);
  CHECK(stub::calls.num_layers == TL_MAX_COMMIT_LAYERS);
  CHECK(stub::calls.last_layer_state == F<float>(0x100000 + 0x10000 * (uintptr_t)(TL_MAX_COMMIT_LAYERS - 1)));
  std::vector<tl_layer> three(layers.begin(), layers.begin() + 3);
  three.shrink_to_fit();
  CHECK(tree_state_commit_layers(&p, 3, three.data(), F<const int32_t>(0x1000), F<const int32_t>(0x2000),
                                 F<const int32_t>(0x5000), nullptr, nullptr, nullptr) == TL_OK);
  CHECK(stub::calls.num_layers == 3 && stub::calls.unused_layer_state == nullptr);
  CHECK(tree_state_commit_layers(&p, TL_MAX_COMMIT_LAYERS + 1, layers.data(), F<const int32_t>(0x1000),
                                 F<const int32_t>(0x2000), F<const int32_t>(0x5000), nullptr, nullptr,
                                 nullptr) == TL_EINVAL);
  three[2].v = P(0x30008);                                // one misaligned layer fails the call
  const int cl_before = stub::calls.commit_layers;
  CHECK(tree_state_commit_layers(&p, 3, three.data(), F<const int32_t>(0x1000), F<const int32_t>(0x2000),
                                 F<const int32_t>(0x5000), nullptr, nullptr, nullptr) == TL_EINVAL);
  CHECK(stub::calls.commit_layers == cl_before);

  // ---- accepted path, topology
  CHECK(tree_accepted_path(&p, F<const int32_t>(0x1000), F<const int32_t>(0x2000), F<const int32_t>(0x5000),
                           F<int32_t>(0x6000), F<int32_t>(0x7000), nullptr, nullptr) == TL_OK);
  CHECK(stub::calls.path == 1);
  tl_problem pt = problem(4, 2, 4, 128, 200, TL_MODE_GLA);
  CHECK(tree_topology_export(&pt, F<const int32_t>(0x1000), F<const int32_t>(0x2000), F<uint64_t>(0x8000),
                             F<int32_t>(0x9000), nullptr, nullptr) == TL_OK);
  CHECK(stub::calls.topo_words == 4);
  CHECK(tree_topology_export(&pt, F<const int32_t>(0x1000), F<const int32_t>(0x2000), F<uint64_t>(0x8004),
                             F<int32_t>(0x9000), nullptr, nullptr) == TL_EINVAL);

  // ---- convolution front end
  tl_problem pc = problem(32, 16, 32, 128, 64, TL_MODE_GDN);
  CHECK(tree_conv_gates(&pc, 4, 1e-6f, F<const int32_t>(0x1000), F<const int32_t>(0x2000), P(0x10000),
                        F<const float>(0x3000), F<const float>(0x3100), F<const float>(0x40000),
                        F<const float>(0x50000), F<const float>(0x3200), F<const float>(0x3300), P(0x60000),
                        nullptr, P(0x70000), P(0x80000), P(0x90000), F<float>(0xa000), F<float>(0xb000),
                        nullptr, nullptr) == TL_OK);
  CHECK(stub::calls.conv == 1 && stub::calls.conv_channels == 2 * 16 * 128 + 32 * 128);
  CHECK(stub::calls.conv_width == 4 && stub::calls.conv_gdn);
  CHECK(tree_conv_state_commit(&pc, 3, F<const int32_t>(0x1000), F<const int32_t>(0x2000),
                               F<const int32_t>(0x5000), P(0x10000), P(0x60000), nullptr, nullptr,
                               nullptr) == TL_OK);
  CHECK(stub::calls.conv_commit_tiles == (8192 + 2047) / 2048);

  // ---- budget allocation, with a caller workspace
  tl_problem pb = problem(128, 1, 1, 16, 256, TL_MODE_GLA);
  const size_t need = tree_budget_workspace_bytes(128, 256);
  CHECK(need > 0 && need % 256 == 0);
  auto budget = [&](const tl_problem* q, void* ws, size_t bytes) {
    return tree_budget_select(q, 20000, 8192, F<const int32_t>(0x1000), F<const int32_t>(0x2000),
                              F<const float>(0x3000), F<float>(0x4000), F<int32_t>(0x5000),
                              F<int32_t>(0x6000), F<int32_t>(0x7000), F<int32_t>(0x8000), ws, bytes,
                              nullptr, nullptr);
  };
  CHECK(budget(&pb, P(0x1000000), need - 1) == TL_EINVAL);
  CHECK(budget(&pb, P(0x1000010), need) == TL_EINVAL);
  CHECK(budget(&pb, P(0x1000000), need) == TL_OK);
  {
    const tl::BudgetArgs& a = stub::calls.budget_args;
    const uintptr_t lo = 0x1000000, hi = lo + need;
    auto inside = [&](const void* x, size_t n) {
      return (uintptr_t)x >= lo && (uintptr_t)x + n <= hi;
    };
    CHECK(inside(a.ws_meta, 128 * 16) && inside(a.ws_key, 128 * 256 * 4));
    CHECK(inside(a.ws_cand, 128 * 256 * 4) && inside(a.ws_root, 128 * 256 * 2));
    CHECK(a.capacity == 8192 && a.num_candidates == 20000 && a.max_nodes == 256);
  }
  // ---- budget allocation without a workspace: refused beyond the static
  // buffer before any lookup; otherwise the static buffer is used
  const int lookups = stub::calls.scratch;
  tl_problem big = problem(408, 1, 1, 16, 256, TL_MODE_GLA);
  auto noalloc = [&](const tl_problem* q) {
    return tree_budget_select_noalloc(q, 20000, 8192, F<const int32_t>(0x1000), F<const int32_t>(0x2000),
                                      F<const float>(0x3000), F<float>(0x4000), F<int32_t>(0x5000),
                                      F<int32_t>(0x6000), F<int32_t>(0x7000), F<int32_t>(0x8000), nullptr,
                                      nullptr);
  };
  CHECK(noalloc(&big) == TL_EUNSUPPORTED);
  CHECK(stub::calls.scratch == lookups);
  stub::calls.scratch_base = P(0x2000000);
  CHECK(noalloc(&pb) == TL_OK);
  CHECK(stub::calls.scratch == lookups + 1);
  CHECK((uintptr_t)stub::calls.budget_args.ws_meta == 0x2000000);
  CHECK((uintptr_t)stub::calls.budget_args.ws_root + 128 * 256 * 2 <= 0x2000000 + TL_BUDGET_NOALLOC_MAX_BYTES);

  if (failures) {
    std::fprintf(stderr, "%d check(s) failed\n", failures);
    return 1;
  }
  std::printf("abi driver: all checks held\n");
  return 0;
}
