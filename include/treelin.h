/*
 * treelin — tree-parallel verification and accepted-path commit for recurrent
 * linear-attention layers (gated linear attention and the gated delta rule)
 * over a drafted token tree, on AMD Instinct MI355X (gfx950).
 *
 * The method follows "Bole: Efficient Tree Speculation for Hybrid-Attention
 * Language Models" (arXiv 2608.01651):
 *   - sequential rule and notation: §4.1, Table "Notation for closed-form tree
 *     verification", restating §2.1 Eq. (gdn-background) node-wise;
 *   - verify = Theorem 1 of §4.1, Eq. (main-closed-form), built from Lemma 1
 *     (Eq. path-factorization / factorized-readout) and Lemma 2
 *     (Eq. correction-system); value tiling as in §4.2 Eq. (kernel-dataflow);
 *   - commit = §4.4 Eq. (accepted-commit) over the accepted path;
 *   - forest layout: §5.2 (flat-ragged forest, request offsets + parents).
 *
 * Conventions used by every entry point
 * -------------------------------------
 * Requests.  A batch of B requests forms a flat-ragged forest.  Request b owns
 *   global rows node_offsets[b] .. node_offsets[b+1]-1 of every per-node array;
 *   T_b = node_offsets[b+1] - node_offsets[b] is its node count.
 * Trees.  parent[r] is request-local: -1 means the node reads the committed
 *   prefix state S_pre (the paper's pi(i) = 0 with S_0 = S_pre); otherwise
 *   0 <= parent < the node's own local index (parent-before-child order).
 *   Several roots per request are allowed.
 * Heads.  Hk query/key heads, Hv value/state heads (Hv a multiple of Hk);
 *   v-head h reads q/k head h / (Hv/Hk).
 * Gates.  g[r, h] is the log-decay (gamma = exp(g), g <= 0 in practice);
 *   beta[r, h] is the delta rule's write gate.
 * State.  One slot per request per layer in the canonical [Hv, d_v, d_k]
 *   layout of §4.4: state[s, h, a, c] is row a (value channel), column c (key
 *   channel) of the paper's S^T.  A node's output is o = q_scale * S_i^T q_i.
 *   Gated linear attention:  S_i = gamma_i S_parent + k_i v_i^T.
 *   Gated delta rule:        u_i = beta_i (v_i - gamma_i S_parent^T k_i),
 *                            S_i = gamma_i S_parent + k_i u_i^T.
 * Layouts (all row-major, contiguous, caller-owned DEVICE memory):
 *   q, k     [N, Hk, d_k]  bf16 or fp32 (tl_problem.in_dtype)
 *   v        [N, Hv, d_v]  same dtype as q, k
 *   g, beta  [N, Hv]       fp32
 *   state    [num_slots, Hv, d_v, d_k] fp32
 *   out      [N, Hv, d_v]  fp32
 *   N = node_offsets[B] rows; ints are int32.
 * Alignment.  q, k, v, state and out must be 16-byte aligned; every other
 *   pointer 4-byte aligned.
 * Streams.  `stream` is a hipStream_t (NULL = the null stream).  Every entry
 *   point only enqueues work on it and returns; results are ready once the
 *   stream has been synchronised.  The library allocates nothing, keeps no
 *   global state and is safe to call from several threads.
 * Errors.  Problems visible from the host (null or misaligned pointers,
 *   unsupported sizes) return a status synchronously and enqueue nothing.
 *   Problems only visible in device data are reported through *dev_err (may
 *   be NULL): the first failing request stores its code there (compare-and-
 *   swap from 0; the caller zeroes it beforehand) and that request is skipped
 *   -- verify leaves its output rows unwritten, commit leaves its slot
 *   untouched.  Other requests are processed normally.
 */
#ifndef TREELIN_H
#define TREELIN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TL_OK = 0,
  TL_EINVAL = 1,       /* bad argument: null/misaligned pointer, bad counts, bad slot */
  TL_EBADTREE = 2,     /* decreasing node_offsets, T_b > max_nodes, or a bad parent */
  TL_EBADPATH = 3,     /* accepted path is not a root-first chain of the request's tree */
  TL_EUNSUPPORTED = 4, /* head dims or max_nodes outside what the kernels implement */
  TL_EHIP = 5          /* the HIP runtime refused a launch */
} tl_status;

typedef enum { TL_MODE_GLA = 0, TL_MODE_GDN = 1 } tl_mode;
typedef enum { TL_BF16 = 0, TL_F32 = 1 } tl_dtype;

typedef struct tl_problem {
  int32_t batch;        /* B >= 0 requests; 0 is a no-op */
  int32_t num_qk_heads; /* Hk >= 1 */
  int32_t num_v_heads;  /* Hv >= 1, a multiple of Hk */
  int32_t d_k;          /* key channels per head: 16, 32, 64 or 128 */
  int32_t d_v;          /* value channels per head: equal to d_k */
  int32_t max_nodes;    /* bound on every T_b, 1..256 (sizes on-chip buffers) */
  int32_t num_slots;    /* slots in `state`; >= B when `slot` is NULL */
  int32_t mode;         /* tl_mode */
  int32_t in_dtype;     /* tl_dtype of q, k, v */
  float q_scale;        /* multiplies every output (1.0f: none) */
} tl_problem;

/* Bytes of layer-local device workspace that tree_lin_attn_verify needs for
 * `problem` (the scratch whose lifetime is one layer's verification, the
 * shortest of the three lifetimes of §4.4; §4.2 keeps the factors C, G and U
 * of Eq. kernel-dataflow inside the tile's workgroup).  Every kernel of this
 * library keeps those factors, the masks and the decays in registers and
 * LDS, so the size is 0 for every problem the library supports; a caller
 * should still size its buffer with this call.  Returns 0 for a NULL or
 * invalid problem as well. */
size_t tl_workspace_bytes(const tl_problem* problem);

/* Tree-parallel verification (Theorem 1 of §4.1, value-tiled as in §4.2).
 *
 * For every node i of every request, writes
 *   out[i, h, :] = q_scale * S_i^T q_i
 * where S_i is the state that sequential execution of the recurrence along
 * the node's root path would produce from S_pre = state[slot(b), h]; no such
 * per-node state is ever formed.  `beta` must be NULL for TL_MODE_GLA and
 * non-NULL for TL_MODE_GDN.  `slot` maps request -> state slot ([B] int32,
 * each in [0, num_slots)); NULL means slot(b) = b.  `state` is only read.
 * workspace: caller-owned device memory of workspace_bytes bytes, at least
 *   tl_workspace_bytes(problem) (TL_EINVAL otherwise); may be NULL when
 *   workspace_bytes is 0; a non-NULL workspace must be 256-byte aligned.
 *   Its contents need no initialisation; calls sharing one must not overlap.
 * Device errors: TL_EBADTREE (forest), TL_EINVAL (slot index). */
tl_status tree_lin_attn_verify(const tl_problem* problem,
                               const int32_t* node_offsets, /* [B+1] */
                               const int32_t* parent,       /* [N] */
                               const void* q, const void* k, const void* v,
                               const float* g, const float* beta,
                               const float* state, const int32_t* slot,
                               float* out, int32_t* dev_err,
                               void* workspace, size_t workspace_bytes,
                               void* stream);

/* Accepted-path commit (§4.4 Eq. accepted-commit).
 *
 * For each request b with a non-empty accepted path, overwrites
 * state[slot(b), h] in place with the post-update state of the path's
 * terminal node, replaying the path in fp32 from the slot's current
 * contents.  path_offsets is [B+1] (non-decreasing, path_offsets[0] = 0) and
 * path[path_offsets[b] .. path_offsets[b+1]-1] lists the accepted nodes,
 * request-local, root first: path[0] is a root and each later entry is a
 * child of the one before.  An empty path leaves the slot untouched (no
 * token accepted keeps S_pre).  Enqueue after the verify that reads the same
 * slots, on the same stream.  Requests naming the same slot race.
 * Device errors: TL_EBADTREE (forest), TL_EBADPATH (path), TL_EINVAL (slot,
 * or decreasing path_offsets). */
tl_status tree_state_commit(const tl_problem* problem,
                            const int32_t* node_offsets, const int32_t* parent,
                            const int32_t* path_offsets, /* [B+1] */
                            const int32_t* path,         /* [path_offsets[B]] */
                            const void* k, const void* v,
                            const float* g, const float* beta,
                            float* state, const int32_t* slot,
                            int32_t* dev_err, void* stream);

/* One recurrent layer's inputs to tree_state_commit_layers: the same rows and
 * layouts as tree_state_commit's k, v, g, beta and state (device pointers;
 * beta NULL for TL_MODE_GLA, non-NULL for TL_MODE_GDN). */
typedef struct tl_layer {
  const void* k;      /* [N, Hk, d_k] */
  const void* v;      /* [N, Hv, d_v] */
  const float* g;     /* [N, Hv] */
  const float* beta;  /* [N, Hv] or NULL */
  float* state;       /* [num_slots, Hv, d_v, d_k], updated in place */
} tl_layer;

/* Most layers one tree_state_commit_layers call takes. */
#define TL_MAX_COMMIT_LAYERS 64

/* Unified cross-layer commit (§5.2 "Unified cross-layer state commit", with
 * §4.4 Eq. accepted-commit per layer).
 *
 * The accepted path is shared by every recurrent layer, so the commits of
 * num_layers layers (0 .. TL_MAX_COMMIT_LAYERS; 0 does nothing) are enqueued
 * by one call: as one launch while a layer's B * Hv slots are fewer than the
 * GPU holds at once, else as one launch per layer (a layer that fills the
 * GPU on its own streams faster alone).  The path
 * of request b is given by its sampled terminal node: terminal[b] is a
 * request-local node index, or -1 when no draft token was accepted (every
 * layer's slot keeps S_pre).  The path is that node and its ancestors, root
 * first, and each layer's slot is updated exactly as tree_state_commit
 * would update it with that path (bit-identical results).  `layers` is a
 * HOST array of num_layers entries, read before the call returns; all
 * layers share the forest, the slot map and the problem's shape.  Layers
 * naming the same state memory race.
 * Device errors: TL_EBADTREE (forest), TL_EBADPATH (terminal < -1 or >= T_b),
 * TL_EINVAL (slot index). */
tl_status tree_state_commit_layers(const tl_problem* problem, int32_t num_layers,
                                   const tl_layer* layers,
                                   const int32_t* node_offsets, const int32_t* parent,
                                   const int32_t* terminal, /* [B] */
                                   const int32_t* slot, int32_t* dev_err, void* stream);

/* Device path compaction (§5.2): the accepted path of every request from its
 * sampled terminal node, for consumers that need the accepted rows (e.g. the
 * attention layers' cache commit, or tree_state_commit's path argument after
 * a prefix sum of path_len).  Writes path_len[b] (0 when terminal[b] == -1)
 * and the path's request-local nodes, root first, at
 * path[node_offsets[b] + t] for t < path_len[b]; the request's other entries
 * of `path` are left as they are.  Device errors: TL_EBADTREE (forest),
 * TL_EBADPATH (terminal < -1 or >= T_b); nothing of that request is
 * written. */
tl_status tree_accepted_path(const tl_problem* problem,
                             const int32_t* node_offsets, const int32_t* parent,
                             const int32_t* terminal, /* [B] */
                             int32_t* path_len,       /* [B] */
                             int32_t* path,           /* [N] */
                             int32_t* dev_err, void* stream);

/* Tree-parallel convolution front end (§4.3 "Stage 1: tree-parallel
 * convolution and gate preparation"; the convolution and gates of §2.1).
 *
 * For every node i, with C = 2 Hk d_k + Hv d_v channels and w = conv_width
 * (2..4):
 *   y_i[c] = conv_bias[c] + sum_{p<w} conv_weight[c, p] * s_i[p][c]
 * where s_i is the last w rows of (the request's convolution state rows,
 * then the x rows of the node's root path, root first): p = w-1 is node i,
 * p = w-2 its parent, and above the root the window continues into the
 * committed state.  z = y * sigmoid(y) (SiLU) is split into q | k | v; q
 * and k are normalised per head, z / sqrt(sum z^2 + norm_eps), and all three
 * are stored as bf16 (round to nearest even).  Gates per (node, v-head):
 *   g = -exp(A_log[h]) * softplus(gate_a + dt_bias[h])   (the log-decay
 *       tree_lin_attn_verify takes),
 *   beta = sigmoid(gate_b)                               (delta rule only).
 * The arithmetic is fp32.
 * Layouts: x [N, C] bf16 (channels q | k | v, head-major); gate_a, gate_b
 *   [N, Hv] fp32; conv_weight [C, w] fp32; conv_bias [C] fp32; A_log,
 *   dt_bias [Hv] fp32; conv_state [num_slots, w-1, C] bf16, rows oldest
 *   first; outputs q, k [N, Hk, d_k], v [N, Hv, d_v] bf16, g, beta [N, Hv]
 *   fp32.  problem->in_dtype must be TL_BF16.  gate_b and beta are NULL for
 *   TL_MODE_GLA and non-NULL for TL_MODE_GDN.  x, conv_state, q, k, v,
 *   conv_weight and conv_bias must be 16-byte aligned.
 * Device errors: TL_EBADTREE (forest), TL_EINVAL (slot index); that
 * request's rows are left unwritten. */
tl_status tree_conv_gates(const tl_problem* problem, int32_t conv_width, float norm_eps,
                          const int32_t* node_offsets, const int32_t* parent,
                          const void* x, const float* gate_a, const float* gate_b,
                          const float* conv_weight, const float* conv_bias,
                          const float* A_log, const float* dt_bias,
                          const void* conv_state, const int32_t* slot,
                          void* q, void* k, void* v, float* g, float* beta,
                          int32_t* dev_err, void* stream);

/* Convolution-state commit: the state of request b becomes the last w-1 rows
 * of (its state rows, the x rows of the accepted path ending at terminal[b],
 * root first), written in place; terminal -1 leaves it untouched.  Enqueue
 * after the tree_conv_gates call that reads the same slots.  The rows are
 * copied exactly (bf16).  Device errors: TL_EBADTREE, TL_EBADPATH (terminal
 * outside [-1, T_b)), TL_EINVAL (slot index); that slot is left untouched. */
tl_status tree_conv_state_commit(const tl_problem* problem, int32_t conv_width,
                                 const int32_t* node_offsets, const int32_t* parent,
                                 const int32_t* terminal, const void* x,
                                 void* conv_state, const int32_t* slot,
                                 int32_t* dev_err, void* stream);

/* Batch-wide verification-budget allocation and forest materialiser (§5.1
 * "Batch-wide utility allocation"; the packed forest of §5.2).
 *
 * Input: per request b a drafter's candidate tree of M_b nodes (parents
 * before children, -1 for a root) with the draft probability p(u | parent(u))
 * of every node, in [0, 1].  Computes
 *   rho(v) = p(root) * ... * p(v) along v's root path, in fp32, root first,
 *            one rounding per step;
 *   rank(v) = v's position among its request's non-root candidates in the
 *            order (rho descending, index ascending); -1 for roots.
 * Every root is kept; K = capacity - (all roots) further nodes are the first
 * K eligible candidates of the batch in the order (rho descending, batch-wide
 * index ascending), where a candidate is eligible while rank(v) <
 * max_nodes - (roots of its request), so no request exceeds max_nodes.  The
 * selected nodes of each request form a prefix-connected subtree; they are
 * packed request by request in candidate order:
 *   node_offsets [B+1]: the per-request budgets' exclusive scan (sum <= capacity);
 *   parent [N]: request-local parent of each packed node in packed numbering;
 *   src [N]: batch-wide candidate index of each packed node,
 * so that node_offsets and parent are tree_lin_attn_verify's forest and src
 * gathers its per-node rows.  Entries past node_offsets[B] are not written.
 * Layouts: cand_offsets [B+1] (cand_offsets[0] = 0, non-decreasing,
 *   cand_offsets[B] <= num_candidates), cand_parent [num_candidates] int32
 *   request-local, cand_prob [num_candidates] fp32; rho, rank
 *   [num_candidates]; parent, src [capacity].  Only batch and max_nodes of
 *   `problem` are used (the rest is checked as for tree_lin_attn_verify).
 * workspace: caller-owned device memory of at least
 *   tree_budget_workspace_bytes(B, max_nodes) bytes, 256-byte aligned; its
 *   contents need no initialisation and are overwritten (calls that share a
 *   workspace must not overlap).
 * Bounds: B <= 1024, M_b <= 1024, num_candidates <= 32768 (TL_EUNSUPPORTED
 *   on the host; a device size beyond them is TL_EINVAL).
 * Device errors: TL_EBADTREE (offsets), TL_EINVAL (a request with more than
 *   1024 candidates or more roots than max_nodes, capacity below the roots):
 *   nothing is selected and node_offsets is all zero.  Per request,
 *   TL_EBADTREE (a bad parent) or TL_EINVAL (a probability outside [0, 1]):
 *   that request keeps only its roots, its rho and rank are unspecified. */
tl_status tree_budget_select(const tl_problem* problem, int32_t num_candidates, int32_t capacity,
                             const int32_t* cand_offsets, const int32_t* cand_parent,
                             const float* cand_prob,
                             float* rho, int32_t* rank,     /* [num_candidates] out */
                             int32_t* node_offsets,         /* [B+1] out */
                             int32_t* parent, int32_t* src, /* [capacity] out */
                             void* workspace, size_t workspace_bytes,
                             int32_t* dev_err, void* stream);

/* Bytes of tree_budget_select's workspace for a batch of `batch` requests
 * and a per-request bound of `max_nodes` nodes (0 for an empty batch). */
size_t tree_budget_workspace_bytes(int32_t batch, int32_t max_nodes);

/* Largest workspace tree_budget_select_noalloc can serve: 1 MiB, i.e.
 * tree_budget_workspace_bytes(batch, max_nodes) <= this, which holds e.g. for
 * batch <= 1024 at max_nodes <= 100 and batch <= 407 at max_nodes = 256. */
#define TL_BUDGET_NOALLOC_MAX_BYTES (1u << 20)

/* tree_budget_select without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments, results and errors as
 * tree_budget_select minus workspace and workspace_bytes: the workspace is a
 * static device array of TL_BUDGET_NOALLOC_MAX_BYTES bytes inside the
 * library, one per GPU, held until the process ends.  Nothing is allocated
 * on any call (the first call on a device looks up that device's array).
 * A problem whose workspace would exceed it returns TL_EUNSUPPORTED before
 * anything is enqueued.  Every call on one GPU shares that GPU's array, so
 * calls that overlap on one GPU (several streams, several threads) race;
 * calls on one stream are ordered and safe.  The array needs no clearing:
 * each call writes every entry it later reads. */
tl_status tree_budget_select_noalloc(const tl_problem* problem, int32_t num_candidates,
                                     int32_t capacity,
                                     const int32_t* cand_offsets, const int32_t* cand_parent,
                                     const float* cand_prob,
                                     float* rho, int32_t* rank,     /* [num_candidates] out */
                                     int32_t* node_offsets,         /* [B+1] out */
                                     int32_t* parent, int32_t* src, /* [capacity] out */
                                     int32_t* dev_err, void* stream);

/* Tree topology of §4.1's notation table, as the kernels build it:
 * anc_mask[r, w] (W = ceil(max_nodes/64) uint64 words per node) has bit
 * (j mod 64) of word j/64 set iff local node j is r's node itself or one of
 * its ancestors (the row of M+ = M- + I); depth[r] is the number of strict
 * ancestors (a root has depth 0).  Device errors: TL_EBADTREE; rows of a
 * malformed request are left unwritten. */
tl_status tree_topology_export(const tl_problem* problem,
                               const int32_t* node_offsets, const int32_t* parent,
                               uint64_t* anc_mask, /* [N, W] */
                               int32_t* depth,     /* [N] */
                               int32_t* dev_err, void* stream);

/* Static, human-readable name of a status code. */
const char* tl_status_string(tl_status status);

/* Library version as "major.minor.patch". */
const char* tl_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TREELIN_H */
