"""fp64 CPU oracle for tree-parallel verification and accepted-path commit of
recurrent linear-attention layers (gated linear attention and the gated delta
rule) over a drafted token tree.

TEST INFRASTRUCTURE ONLY.  Nothing in the library imports this module.  It may
be imported only by the tests, by the smoke check and by the CPU-baseline leg
of the benchmark.  It shares no code with the HIP path.

What is computed, and where the paper defines it
------------------------------------------------
* Sequential rule (paper §2.1 Eq. gdn-background, restated node-wise in §4.1,
  Table "Notation for closed-form tree verification"): node i starts from its
  parent's post-update state S_pi(i) (S_pre for a root), decays it by gamma_i,
  applies its own update, and reads the post-update state out with q_i.
* Verify = that sequential tree execution, done branch by branch: for every
  node the recurrence is re-run from S_pre along the node's own root-to-node
  path (no memoised parent states).  Theorem 1 of §4.1 states that the closed
  form equals exactly this, and §4.1 shows its solution is unique, so the
  definition is what the oracle computes.
* Commit = the post-update state at the accepted terminal node (Lemma 1 with
  Eq. accepted-commit in §4.4), i.e. the same walk over the accepted path; an
  empty path leaves S_pre unchanged (end of §4.4).

Conventions (readings of the paper; the kernels take the same ones)
------------------------------------------------------------------------------
* Stored state orientation: the paper's state is S in R^{d_k x d_v} with
  o = S^T q; slots use the canonical [H, d_v, d_k] layout (§4.4).  The oracle
  keeps the stored matrix St = S^T of shape [d_v, d_k], so o = St @ q and the
  GLA update is St <- gamma*St + outer(v, k).
* Nodes are 0-based and request-local; parent -1 means "reads S_pre" (the
  paper's pi(i)=0 with S_0=S_pre); every other parent is smaller than the node
  (parent-before-child ordering, §4.1).
* gamma = exp(g) with g the fp32 log-decay per (node, v-head); beta per
  (node, v-head) for the delta rule.
* GQA: v-head h reads qk-head h // (Hv // Hk).
* Outputs are scaled by q_scale (1.0 in every workload).

Parity pins: see tests/test_oracle_pins.py.  The GQA head grouping and q_scale
are conventions the paper does not fix; both sides take the same reading of
each.  The oracle's implementation of the two is pinned against their
definitions: grouped heads equal the ungrouped computation on qk-heads repeated
in place (numpy.repeat), and q_scale equals scaling the queries.
"""
from __future__ import annotations

import numpy as np

GLA = 0
GDN = 1
BF16 = 0
F32 = 1

MAX_NODES_LIMIT = 256
SUPPORTED_D = (16, 32, 64, 128)


class OracleError(Exception):
    """Base class; the status code mirrors the C ABI's tl_status values."""
    status = 0


class InvalidArg(OracleError):
    status = 1


class BadTree(OracleError):
    status = 2


class BadPath(OracleError):
    status = 3


class Unsupported(OracleError):
    status = 4


# --------------------------------------------------------------------------
# argument checks (mirrors the library's synchronous and device checks)
# --------------------------------------------------------------------------

def check_problem(batch, num_qk_heads, num_v_heads, d_k, d_v, max_nodes, mode):
    if batch < 0 or num_qk_heads <= 0 or num_v_heads <= 0:
        raise InvalidArg("batch/head counts out of range")
    if num_v_heads % num_qk_heads:
        raise InvalidArg("num_v_heads must be a multiple of num_qk_heads")
    if mode not in (GLA, GDN):
        raise InvalidArg("unknown mode")
    if d_k not in SUPPORTED_D or d_v not in SUPPORTED_D:
        raise Unsupported("head dims must be one of 16, 32, 64, 128")
    if not (1 <= max_nodes <= MAX_NODES_LIMIT):
        raise Unsupported("max_nodes must lie in [1, 256]")


def check_forest(node_offsets, parent, max_nodes):
    """Flat-ragged forest (§5.2): request b owns rows
    node_offsets[b] .. node_offsets[b+1]-1 of every per-node tensor.
    Raises InvalidArg for arrays of the wrong shape and BadTree for a forest
    that is not well formed: decreasing offsets, a request larger than
    max_nodes, or a parent that breaks the parent-before-child ordering of
    §4.1 (the library reports the same three cases as TL_EBADTREE)."""
    node_offsets = np.asarray(node_offsets, dtype=np.int64)
    parent = np.asarray(parent, dtype=np.int64)
    if node_offsets.ndim != 1 or node_offsets.size < 1 or node_offsets[0] != 0:
        raise InvalidArg("node_offsets must start at 0")
    sizes = np.diff(node_offsets)
    if np.any(sizes < 0):
        raise BadTree("node_offsets must be non-decreasing")
    if np.any(sizes > max_nodes):
        raise BadTree("a request has more than max_nodes nodes")
    if node_offsets[-1] != parent.size:
        raise InvalidArg("parent length must equal node_offsets[-1]")
    for b in range(sizes.size):
        p = parent[node_offsets[b]:node_offsets[b + 1]]
        for i, pi in enumerate(p):
            if not (pi == -1 or 0 <= pi < i):
                raise BadTree(f"request {b}: parent[{i}]={pi} is not -1 or in [0,{i})")


def check_paths(node_offsets, parent, path_offsets, path):
    """Accepted path of §4.4: P(a) = Anc(a) u {a}, listed root first."""
    node_offsets = np.asarray(node_offsets, dtype=np.int64)
    path_offsets = np.asarray(path_offsets, dtype=np.int64)
    path = np.asarray(path, dtype=np.int64)
    B = node_offsets.size - 1
    if path_offsets.size != B + 1 or path_offsets[0] != 0:
        raise InvalidArg("path_offsets must have batch+1 entries starting at 0")
    if np.any(np.diff(path_offsets) < 0) or path_offsets[-1] != path.size:
        raise InvalidArg("path_offsets must be non-decreasing and end at len(path)")
    for b in range(B):
        T = node_offsets[b + 1] - node_offsets[b]
        p = path[path_offsets[b]:path_offsets[b + 1]]
        if p.size > T:
            raise BadPath(f"request {b}: path longer than the tree")
        prev = -1
        for a in p:
            if not (0 <= a < T):
                raise BadPath(f"request {b}: path node {a} outside [0,{T})")
            if parent[node_offsets[b] + a] != prev:
                raise BadPath(f"request {b}: path is not a root-first chain")
            prev = a


# --------------------------------------------------------------------------
# topology
# --------------------------------------------------------------------------

def root_path(parent_b, i):
    """Root-first list of Anc(i) u {i} for request-local parent array."""
    out = []
    j = int(i)
    while j != -1:
        out.append(j)
        j = int(parent_b[j])
    out.reverse()
    return out


def topology(node_offsets, parent, max_nodes):
    """Inclusive ancestor masks M+ (§4.1 notation table: M+ = M- + I) as
    ceil(max_nodes/64) little-endian uint64 words per node (bit j of node i's
    row is set iff j is i or an ancestor of i, request-local), and depth =
    number of strict ancestors (a root has depth 0)."""
    check_forest(node_offsets, parent, max_nodes)
    node_offsets = np.asarray(node_offsets, dtype=np.int64)
    parent = np.asarray(parent, dtype=np.int64)
    W = (max_nodes + 63) // 64
    N = parent.size
    mask = np.zeros((N, W), dtype=np.uint64)
    depth = np.zeros(N, dtype=np.int32)
    for b in range(node_offsets.size - 1):
        o = node_offsets[b]
        pb = parent[o:node_offsets[b + 1]]
        for i in range(pb.size):
            path = root_path(pb, i)
            depth[o + i] = len(path) - 1
            for j in path:
                mask[o + i, j // 64] |= np.uint64(1) << np.uint64(j % 64)
    return mask, depth


# --------------------------------------------------------------------------
# the recurrence (stored orientation St = S^T, shape [d_v, d_k])
# --------------------------------------------------------------------------

def step(mode, St, k, v, g, beta):
    """One sequential update of §2.1 Eq. gdn-background, in the stored
    orientation.  St: [..., d_v, d_k]; k: [..., d_k]; v: [..., d_v];
    g, beta: [...].  Returns the post-update state (a new array)."""
    gamma = np.exp(g)[..., None, None]
    St_tilde = gamma * St                                  # S~ = gamma S
    if mode == GLA:
        u = v                                              # plain GLA: u := v
    else:
        pred = np.einsum("...vk,...k->...v", St_tilde, k)  # S~^T k, stored form
        u = beta[..., None] * (v - pred)                   # u = beta (v - S~^T k)
    return St_tilde + u[..., :, None] * k[..., None, :]    # S = S~ + k u^T


def _as_f64(x):
    return None if x is None else np.asarray(x, dtype=np.float64)


def _slot_of(slot, b):
    return b if slot is None else int(slot[b])


def verify(mode, num_qk_heads, node_offsets, parent, q, k, v, g, beta, state,
           slot=None, q_scale=1.0, max_nodes=MAX_NODES_LIMIT):
    """Outputs o_i for every node of every request.

    q, k: [N, Hk, d_k]; v: [N, Hv, d_v]; g, beta: [N, Hv];
    state: [num_slots, Hv, d_v, d_k] (S_pre, stored orientation);
    slot: [B] request -> state slot, or None for identity.
    Returns O: [N, Hv, d_v] float64.

    Each node walks its own root-to-node path from a fresh copy of S_pre
    (sequential tree execution, §4.1), all v-heads at once."""
    q, k, v, g, beta, state = map(_as_f64, (q, k, v, g, beta, state))
    Hv = v.shape[1]
    _check_shapes(mode, num_qk_heads, Hv, q, k, v, g, beta, state, slot,
                  len(node_offsets) - 1, max_nodes)
    check_forest(node_offsets, parent, max_nodes)
    grp = Hv // num_qk_heads
    hq = np.arange(Hv) // grp                  # GQA: v-head h reads qk-head h // grp
    O = np.zeros(v.shape, dtype=np.float64)
    for b in range(len(node_offsets) - 1):
        o = int(node_offsets[b])
        pb = np.asarray(parent[o:int(node_offsets[b + 1])])
        S_pre = state[_slot_of(slot, b)]
        for i in range(pb.size):
            St = S_pre.copy()
            for t in root_path(pb, i):
                r = o + t
                St = step(mode, St, k[r, hq], v[r], g[r],
                          None if beta is None else beta[r])
            O[o + i] = q_scale * np.einsum("hvk,hk->hv", St, q[o + i, hq])
    return O


def commit(mode, num_qk_heads, node_offsets, parent, path_offsets, path, k, v,
           g, beta, state, slot=None, max_nodes=MAX_NODES_LIMIT):
    """New state of every request: S_pre walked along its accepted path
    (root first).  An empty path returns S_pre unchanged.  Returns a new
    [num_slots, Hv, d_v, d_k] float64 array; slots no request names are
    copied through."""
    k, v, g, beta, state = map(_as_f64, (k, v, g, beta, state))
    Hv = v.shape[1]
    _check_shapes(mode, num_qk_heads, Hv, None, k, v, g, beta, state, slot,
                  len(node_offsets) - 1, max_nodes)
    check_forest(node_offsets, parent, max_nodes)
    check_paths(node_offsets, parent, path_offsets, path)
    grp = Hv // num_qk_heads
    hq = np.arange(Hv) // grp
    new = state.copy()
    for b in range(len(node_offsets) - 1):
        o = int(node_offsets[b])
        s = _slot_of(slot, b)
        St = state[s].copy()
        for t in path[int(path_offsets[b]):int(path_offsets[b + 1])]:
            r = o + int(t)
            St = step(mode, St, k[r, hq], v[r], g[r],
                      None if beta is None else beta[r])
        new[s] = St
    return new


def accepted_paths(node_offsets, parent, terminal, max_nodes=MAX_NODES_LIMIT):
    """Accepted path of every request from its sampled terminal node (§4.4:
    P(a) = Anc(a) u {a}, listed root first; §5.2: one path descriptor per
    request).  terminal[b] is request-local; -1 means nothing was accepted
    (an empty path).  Raises BadTree for a malformed forest and BadPath for a
    terminal outside [-1, T_b).  Returns (path_offsets, path) in the packed
    form that commit() takes."""
    check_forest(node_offsets, parent, max_nodes)
    node_offsets = np.asarray(node_offsets, dtype=np.int64)
    parent = np.asarray(parent, dtype=np.int64)
    B = node_offsets.size - 1
    if len(terminal) != B:
        raise InvalidArg("terminal must have one entry per request")
    offs = [0]
    flat = []
    for b in range(B):
        T = int(node_offsets[b + 1] - node_offsets[b])
        a = int(terminal[b])
        if not (-1 <= a < T):
            raise BadPath(f"request {b}: terminal {a} outside [-1,{T})")
        p = [] if a == -1 else root_path(parent[node_offsets[b]:node_offsets[b + 1]], a)
        flat.extend(p)
        offs.append(len(flat))
    return np.asarray(offs, dtype=np.int64), np.asarray(flat, dtype=np.int64)


def commit_layers(mode, num_qk_heads, node_offsets, parent, terminal, layers,
                  slot=None, max_nodes=MAX_NODES_LIMIT):
    """Unified cross-layer commit (§5.2): every recurrent layer commits the same
    accepted path, the one ending at terminal[b].  layers is a list of
    (k, v, g, beta, state) per layer; returns the list of new states, each
    exactly commit() of that layer over accepted_paths()."""
    path_offsets, path = accepted_paths(node_offsets, parent, terminal, max_nodes)
    return [commit(mode, num_qk_heads, node_offsets, parent, path_offsets, path,
                   k, v, g, beta, state, slot=slot, max_nodes=max_nodes)
            for (k, v, g, beta, state) in layers]


def prefix_state(mode, k, v, g, beta, St0=None):
    """State after running the recurrence along a plain token sequence (a
    chain), starting from St0 (zeros if None).  Used to build S_pre from a
    synthetic prefix.  k: [L, ..., d_k]; v: [L, ..., d_v]; g, beta: [L, ...].
    Leading axis is time; the remaining axes are batched units."""
    k, v, g, beta = map(_as_f64, (k, v, g, beta))
    if St0 is None:
        St = np.zeros(v.shape[1:] + (k.shape[-1],), dtype=np.float64)
    else:
        St = np.array(St0, dtype=np.float64)
    for t in range(k.shape[0]):
        St = step(mode, St, k[t], v[t], g[t], None if beta is None else beta[t])
    return St


def _check_shapes(mode, Hk, Hv, q, k, v, g, beta, state, slot, B, max_nodes):
    if Hk <= 0 or Hv % Hk:
        raise InvalidArg("num_v_heads must be a multiple of num_qk_heads")
    if mode == GDN and beta is None:
        raise InvalidArg("the delta rule needs beta")
    if mode == GLA and beta is not None:
        raise InvalidArg("gated linear attention takes no beta")
    d_k = k.shape[-1]
    d_v = v.shape[-1]
    if mode not in (GLA, GDN):
        raise InvalidArg("unknown mode")
    if not (1 <= max_nodes <= MAX_NODES_LIMIT):
        raise Unsupported("max_nodes must lie in [1, 256]")
    N = v.shape[0]
    if k.shape != (N, Hk, d_k) or (q is not None and q.shape != (N, Hk, d_k)):
        raise InvalidArg("q/k must be [N, Hk, d_k]")
    if g.shape != (N, Hv) or (beta is not None and beta.shape != (N, Hv)):
        raise InvalidArg("g/beta must be [N, Hv]")
    if state.ndim != 4 or state.shape[1:] != (Hv, d_v, d_k):
        raise InvalidArg("state must be [slots, Hv, d_v, d_k]")
    if slot is None:
        if state.shape[0] < B:
            raise InvalidArg("identity slot map needs num_slots >= batch")
    else:
        s = np.asarray(slot)
        if s.shape != (B,) or np.any(s < 0) or np.any(s >= state.shape[0]):
            raise InvalidArg("slot index out of range")
