"""Seeded synthetic inputs for tree-parallel linear-attention verification.

This module only draws random inputs: draft trees, per-node q/k/v/gates,
accepted paths and the tokens of a committed prefix.  It holds none of the
verify/commit arithmetic; the prefix *state* is built from these tokens by
whoever consumes them (the fp64 oracle in tests, the library's own commit in
the benchmark).

Five workloads, shaped like the paper's evaluation (§6.1: Qwen3.5 GDN layers
with d_k = d_v = 128, draft trees from a top-k = 4, depth-8 drafter, batches of
1-16 requests):

  tiny        1 request, 1 head, d=16, GLA, fp32 q/k/v, complete binary tree
              of depth 3 (15 nodes), S_pre ~ N(0, 0.1^2), one root-to-leaf path.
  mid         1 request, 8 heads, d=128, GLA, bf16, 512-token prefix, 64-node
              rho-selected tree (branching 4,4,2,1,..., depth <= 8), L ~ U{1..8}.
  production  32 requests, 16 qk / 32 v heads, d=128, GLA, bf16, 2048-token
              prefix, 64-node trees (8,4,2,1,..., depth <= 10),
              g = -softplus(N(0,1) - 2).
  gdn         16 requests, shapes as production, gated delta rule,
              alpha = exp(-softplus(N(0,1))), beta = sigmoid(N(0,1)),
              128-node trees (16,4,2,1,..., depth <= 12), L <= 12.
  large       128 requests, shapes as production; request 0 is a 16-node
              chain, the rest are random recursive trees of 32..256 nodes
              (depth <= 16, at least one of exactly 256) in creation order.

Random streams: every request draws from numpy's PCG64 seeded with
[seed, config id, step, request, stream], so any request (or any 256-token
chunk of its prefix) can be regenerated on its own.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

GLA = 0
GDN = 1

CONFIG_IDS = {"tiny": 1, "mid": 2, "production": 3, "gdn": 4, "large": 5}

# stream ids inside one request's seed
_S_TREE, _S_Q, _S_K, _S_V, _S_G, _S_BETA, _S_PATH, _S_STATE = range(8)
_S_PREFIX = 1000          # + chunk index
PREFIX_CHUNK = 256


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    mode: int
    in_dtype: str           # "f32" or "bf16"
    batch: int
    num_qk_heads: int
    num_v_heads: int
    d_k: int
    d_v: int
    max_nodes: int
    tree: tuple             # ("binary", depth) | ("topk", T, branching, depth_cap)
                            # | ("recursive", chain_len, Tmin, Tmax, depth_cap)
    gate_shift: float       # g = -softplus(N(0,1) - gate_shift)
    prefix_len: int         # 0: S_pre drawn directly as N(0, 0.1^2)
    path_rule: tuple        # ("leaf",) | ("uniform", L_cap)
    q_scale: float = 1.0


CONFIGS = {
    "tiny": Config("tiny", GLA, "f32", 1, 1, 1, 16, 16, 15,
                   ("binary", 3), 0.0, 0, ("leaf",)),
    "mid": Config("mid", GLA, "bf16", 1, 8, 8, 128, 128, 64,
                  ("topk", 64, (4, 4, 2), 8), 0.0, 512, ("uniform", 8)),
    "production": Config("production", GLA, "bf16", 32, 16, 32, 128, 128, 64,
                         ("topk", 64, (8, 4, 2), 10), 2.0, 2048, ("uniform", 11)),
    "gdn": Config("gdn", GDN, "bf16", 16, 16, 32, 128, 128, 128,
                  ("topk", 128, (16, 4, 2), 12), 0.0, 2048, ("uniform", 12)),
    "large": Config("large", GLA, "bf16", 128, 16, 32, 128, 128, 256,
                    ("recursive", 16, 32, 256, 16), 2.0, 2048, ("uniform", 16)),
}


# --------------------------------------------------------------------------
# number formats
# --------------------------------------------------------------------------

def bf16_bits(x):
    """Round float32 values to bfloat16 (round to nearest, ties to even) and
    return the 16-bit patterns.  NaN stays a quiet NaN with its sign; +-Inf and
    values that round past the largest finite bf16 become +-Inf."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    nan = np.isnan(f)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)).astype(np.uint16)
    r = np.where(nan, ((u >> np.uint64(16)).astype(np.uint16) | np.uint16(0x0040)), r)
    return r.astype(np.uint16)


def bf16_to_f32(bits):
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32)


def round_bf16(x):
    """float32 array whose values are the bf16 (RNE) roundings of x."""
    return bf16_to_f32(bf16_bits(x))


def _softplus(x):
    return np.logaddexp(0.0, x)


def _sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


# --------------------------------------------------------------------------
# trees and paths
# --------------------------------------------------------------------------

def binary_tree(depth):
    T = 2 ** (depth + 1) - 1
    return np.array([-1] + [(i - 1) // 2 for i in range(1, T)], dtype=np.int32)


def topk_tree(rng, T, branching, depth_cap):
    """Candidate tree whose depth-l nodes have branching[l] children (1 past
    the end of the list) down to depth_cap; each sibling group's draft
    probabilities are softmax(N(0,1)).  The path score rho is the product of
    probabilities along the path (the utility of the paper's §5.1 budget
    allocation).  Keep the root and the T-1 best candidates (ties: lower
    depth, then lower candidate index, so a parent always precedes its
    children), then renumber in BFS order."""
    cand_parent = [-1]
    cand_depth = [0]
    cand_rho = [1.0]
    frontier = [0]
    for lvl in range(depth_cap):
        nb = branching[lvl] if lvl < len(branching) else 1
        nxt = []
        for p in frontier:
            z = rng.standard_normal(nb)
            pr = np.exp(z - z.max())
            pr /= pr.sum()
            for c in range(nb):
                cand_parent.append(p)
                cand_depth.append(lvl + 1)
                cand_rho.append(cand_rho[p] * float(pr[c]))
                nxt.append(len(cand_parent) - 1)
        frontier = nxt
    n = len(cand_parent)
    if n < T:
        raise ValueError(f"candidate tree has {n} < {T} nodes")
    order = sorted(range(1, n), key=lambda c: (-cand_rho[c], cand_depth[c], c))
    keep = sorted([0] + order[:T - 1])        # BFS candidate order is preserved
    new_id = {c: i for i, c in enumerate(keep)}
    parent = np.empty(T, dtype=np.int32)
    for c, i in new_id.items():
        p = cand_parent[c]
        if p != -1 and p not in new_id:
            raise AssertionError("selection is not prefix-connected")
        parent[i] = -1 if p == -1 else new_id[p]
    return parent


def recursive_tree(rng, T, depth_cap):
    """Random recursive tree in creation order: node i >= 1 attaches to a
    uniformly chosen existing node whose depth is below depth_cap."""
    parent = np.empty(T, dtype=np.int32)
    depth = np.empty(T, dtype=np.int32)
    parent[0], depth[0] = -1, 0
    open_nodes = [0]
    for i in range(1, T):
        p = open_nodes[int(rng.integers(len(open_nodes)))]
        parent[i], depth[i] = p, depth[p] + 1
        if depth[i] < depth_cap:
            open_nodes.append(i)
    return parent


def chain_tree(T):
    return np.arange(-1, T - 1, dtype=np.int32)


def node_depths(parent):
    d = np.zeros(parent.size, dtype=np.int32)
    for i, p in enumerate(parent):
        d[i] = 0 if p < 0 else d[p] + 1
    return d


def path_to(parent, a):
    out = []
    while a != -1:
        out.append(int(a))
        a = int(parent[a])
    return out[::-1]


def draw_path(rng, parent, rule):
    depth = node_depths(parent)
    if rule[0] == "leaf":
        is_leaf = np.ones(parent.size, dtype=bool)
        is_leaf[parent[parent >= 0]] = False
        leaves = np.flatnonzero(is_leaf)
        return path_to(parent, leaves[int(rng.integers(leaves.size))])
    d_b = int(depth.max())
    L = int(rng.integers(1, min(rule[1], d_b + 1) + 1)) if rule[1] > 0 else 0
    if L == 0:
        return []
    at = np.flatnonzero(depth == L - 1)
    return path_to(parent, at[int(rng.integers(at.size))])


# --------------------------------------------------------------------------
# one workload
# --------------------------------------------------------------------------

@dataclasses.dataclass
class Workload:
    cfg: Config
    seed: int
    step: int
    node_offsets: np.ndarray     # [B+1] int32
    parent: np.ndarray           # [N] int32, request-local
    q: np.ndarray                # [N, Hk, d_k] float32 (bf16-representable for bf16 configs)
    k: np.ndarray                # [N, Hk, d_k]
    v: np.ndarray                # [N, Hv, d_v]
    g: np.ndarray                # [N, Hv] float32 log-decay
    beta: np.ndarray | None      # [N, Hv] float32 (delta rule only)
    path_offsets: np.ndarray     # [B+1] int32
    path: np.ndarray             # [sum L_b] int32, request-local, root first
    state: np.ndarray | None     # [B, Hv, d_v, d_k] float32 when drawn directly

    @property
    def N(self):
        return int(self.node_offsets[-1])

    @property
    def batch(self):
        return self.node_offsets.size - 1


def _rng(seed, cfg, step, b, stream):
    return np.random.default_rng([seed, CONFIG_IDS[cfg.name], step, b, stream])


def _unit_rows(rng, shape, cfg):
    """N(0,1) vectors normalised to unit L2 norm along the last axis (in
    fp64), then stored in the input dtype."""
    x = rng.standard_normal(shape)
    x /= np.linalg.norm(x, axis=-1, keepdims=True)
    return _store(x, cfg)


def _store(x, cfg):
    x = np.asarray(x, dtype=np.float32)
    return round_bf16(x) if cfg.in_dtype == "bf16" else x


def _tree(cfg, rng, b):
    kind = cfg.tree[0]
    if kind == "binary":
        return binary_tree(cfg.tree[1])
    if kind == "topk":
        _, T, branching, cap = cfg.tree
        return topk_tree(rng, T, branching, cap)
    _, chain_len, tmin, tmax, cap = cfg.tree
    if b == 0:
        return chain_tree(chain_len)
    T = tmax if b == 1 else int(rng.integers(tmin, tmax + 1))
    return recursive_tree(rng, T, cap)


def make_request(cfg, seed, step, b):
    """All tree-token inputs of request b (independent of every other request)."""
    Hk, Hv, dk, dv = cfg.num_qk_heads, cfg.num_v_heads, cfg.d_k, cfg.d_v
    parent = _tree(cfg, _rng(seed, cfg, step, b, _S_TREE), b)
    T = parent.size
    q = _unit_rows(_rng(seed, cfg, step, b, _S_Q), (T, Hk, dk), cfg)
    k = _unit_rows(_rng(seed, cfg, step, b, _S_K), (T, Hk, dk), cfg)
    v = _store(_rng(seed, cfg, step, b, _S_V).standard_normal((T, Hv, dv)), cfg)
    z = _rng(seed, cfg, step, b, _S_G).standard_normal((T, Hv))
    g = (-_softplus(z - cfg.gate_shift)).astype(np.float32)
    beta = None
    if cfg.mode == GDN:
        beta = _sigmoid(_rng(seed, cfg, step, b, _S_BETA).standard_normal((T, Hv))).astype(np.float32)
    path = draw_path(_rng(seed, cfg, step, b, _S_PATH), parent, cfg.path_rule)
    state = None
    if cfg.prefix_len == 0:
        state = (0.1 * _rng(seed, cfg, 0, b, _S_STATE).standard_normal((Hv, dv, dk))).astype(np.float32)
    return dict(parent=parent, q=q, k=k, v=v, g=g, beta=beta,
                path=np.asarray(path, dtype=np.int32), state=state)


def make(cfg, seed=0, step=0, batch=None, requests=None):
    """Workload for config `cfg` (name or Config).  `batch` truncates the
    batch (first requests only); `requests` picks explicit request ids."""
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    if requests is None:
        requests = range(cfg.batch if batch is None else batch)
    reqs = [make_request(cfg, seed, step, b) for b in requests]
    sizes = [r["parent"].size for r in reqs]
    node_offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    plens = [r["path"].size for r in reqs]
    path_offsets = np.concatenate([[0], np.cumsum(plens)]).astype(np.int32)

    def cat(key):
        if reqs and reqs[0][key] is None:
            return None
        return np.concatenate([r[key] for r in reqs]) if reqs else None

    state = None
    if cfg.prefix_len == 0 and reqs:
        state = np.stack([r["state"] for r in reqs])
    Hk, Hv, dk, dv = cfg.num_qk_heads, cfg.num_v_heads, cfg.d_k, cfg.d_v
    empty = lambda *s: np.zeros(s, dtype=np.float32)
    return Workload(
        cfg=cfg, seed=seed, step=step, node_offsets=node_offsets,
        parent=cat("parent") if reqs else np.zeros(0, np.int32),
        q=cat("q") if reqs else empty(0, Hk, dk),
        k=cat("k") if reqs else empty(0, Hk, dk),
        v=cat("v") if reqs else empty(0, Hv, dv),
        g=cat("g") if reqs else empty(0, Hv),
        beta=cat("beta") if cfg.mode == GDN else None,
        path_offsets=path_offsets,
        path=np.concatenate([r["path"] for r in reqs]).astype(np.int32) if reqs else np.zeros(0, np.int32),
        state=state)


def prefix_chunk(cfg, seed, b, chunk):
    """Tokens [chunk*256, (chunk+1)*256) of request b's committed prefix (a
    plain sequence, drawn like the tree tokens).  Returns k [L, Hk, d_k],
    v [L, Hv, d_v], g [L, Hv], beta [L, Hv] or None."""
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    L = min(PREFIX_CHUNK, cfg.prefix_len - chunk * PREFIX_CHUNK)
    if L <= 0:
        raise ValueError("chunk past the end of the prefix")
    rng = _rng(seed, cfg, 0, b, _S_PREFIX + chunk)
    Hk, Hv, dk, dv = cfg.num_qk_heads, cfg.num_v_heads, cfg.d_k, cfg.d_v
    k = _unit_rows(rng, (L, Hk, dk), cfg)
    v = _store(rng.standard_normal((L, Hv, dv)), cfg)
    g = (-_softplus(rng.standard_normal((L, Hv)) - cfg.gate_shift)).astype(np.float32)
    beta = None
    if cfg.mode == GDN:
        beta = _sigmoid(rng.standard_normal((L, Hv))).astype(np.float32)
    return k, v, g, beta


def prefix_chunks(cfg):
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    return math.ceil(cfg.prefix_len / PREFIX_CHUNK)


# --------------------------------------------------------------------------
# inputs of the convolution front end (drawn values only)
# --------------------------------------------------------------------------
_S_CONV_X, _S_CONV_GA, _S_CONV_GB, _S_CONV_STATE = range(20, 24)
_S_CONV_PARAMS = 30


@dataclasses.dataclass
class ConvInputs:
    width: int
    x: np.ndarray                  # [N, C] float32, bf16-representable; C = 2 Hk d_k + Hv d_v
    gate_a: np.ndarray             # [N, Hv] float32 (decay gate pre-activation)
    gate_b: np.ndarray | None      # [N, Hv] float32 (write gate pre-activation; delta rule)
    conv_weight: np.ndarray        # [C, width] float32
    conv_bias: np.ndarray          # [C] float32
    A_log: np.ndarray              # [Hv] float32
    dt_bias: np.ndarray            # [Hv] float32
    conv_state: np.ndarray         # [B, width - 1, C] float32, bf16-representable


def make_conv(w, width=4, requests=None):
    """Front-end inputs over the forest of workload w: per request (seeded by
    request id, like the tree tokens) the mixed projection rows x ~ N(0,1),
    the gate pre-activations ~ N(0,1) and the committed convolution state
    rows ~ N(0,1); per layer the convolution weights ~ N(0, 1/width), bias
    ~ N(0, 0.1^2), A_log = log U(1, 16) and dt_bias = inverse softplus of
    dt = exp U(log 1e-3, log 1e-1) (the usual Gated DeltaNet initialisation)."""
    cfg = w.cfg
    Hk, Hv, dk, dv = cfg.num_qk_heads, cfg.num_v_heads, cfg.d_k, cfg.d_v
    C = 2 * Hk * dk + Hv * dv
    requests = list(range(w.batch)) if requests is None else list(requests)
    assert len(requests) == w.batch
    xs, gas, gbs, sts = [], [], [], []
    for i, b in enumerate(requests):
        T = int(w.node_offsets[i + 1] - w.node_offsets[i])
        xs.append(_rng(w.seed, cfg, w.step, b, _S_CONV_X).standard_normal((T, C)))
        gas.append(_rng(w.seed, cfg, w.step, b, _S_CONV_GA).standard_normal((T, Hv)))
        gbs.append(_rng(w.seed, cfg, w.step, b, _S_CONV_GB).standard_normal((T, Hv)))
        sts.append(_rng(w.seed, cfg, w.step, b, _S_CONV_STATE).standard_normal((width - 1, C)))
    prm = _rng(w.seed, cfg, 0, 0, _S_CONV_PARAMS)
    dt = np.exp(prm.uniform(math.log(1e-3), math.log(1e-1), Hv))
    f32 = lambda a: np.asarray(a, dtype=np.float32)
    cat = lambda parts, cols: np.concatenate(parts) if parts else np.zeros((0, cols))
    return ConvInputs(
        width=width,
        x=round_bf16(f32(cat(xs, C))),
        gate_a=f32(cat(gas, Hv)),
        gate_b=f32(cat(gbs, Hv)) if cfg.mode == GDN else None,
        conv_weight=f32(prm.standard_normal((C, width)) / math.sqrt(width)),
        conv_bias=f32(0.1 * prm.standard_normal(C)),
        A_log=f32(np.log(prm.uniform(1.0, 16.0, Hv))),
        dt_bias=f32(dt + np.log(-np.expm1(-dt))),
        conv_state=round_bf16(f32(np.stack(sts))) if sts else np.zeros((0, width - 1, C), np.float32))


# --------------------------------------------------------------------------
# candidate trees with draft probabilities (inputs of the budget allocation)
# --------------------------------------------------------------------------
_S_CAND = 50


def candidate_tree(rng, branching, depth_cap, quantum=None):
    """A drafter's candidate tree in BFS order: depth-l nodes get branching[l]
    children (1 past the end of the list) down to depth_cap; each sibling
    group's draft probabilities are softmax(N(0,1)), rounded to multiples of
    `quantum` (at least one quantum) when given, so that equal path scores
    occur.  The root's probability is 1.  Returns (parent int32, prob
    float32)."""
    parent, prob, frontier = [-1], [1.0], [0]
    for lvl in range(depth_cap):
        nb = branching[lvl] if lvl < len(branching) else 1
        nxt = []
        for p in frontier:
            z = rng.standard_normal(nb)
            pr = np.exp(z - z.max())
            pr /= pr.sum()
            if quantum:
                pr = np.maximum(np.round(pr / quantum), 1.0) * quantum
            for c in range(nb):
                parent.append(p)
                prob.append(float(pr[c]))
                nxt.append(len(parent) - 1)
        frontier = nxt
    return np.asarray(parent, np.int32), np.asarray(prob, np.float32)


def make_candidates(seed, sizes, quantum=None):
    """A batch of candidate trees: sizes[b] = (branching, depth_cap), or None
    for a request with no candidates.  Returns cand_offsets [B+1], parent [M],
    prob [M]."""
    parents, probs = [], []
    for b, spec in enumerate(sizes):
        if spec is None:
            parents.append(np.zeros(0, np.int32))
            probs.append(np.zeros(0, np.float32))
            continue
        rng = np.random.default_rng([seed, 0, 0, b, _S_CAND])
        p, q = candidate_tree(rng, spec[0], spec[1], quantum)
        parents.append(p)
        probs.append(q)
    offs = np.concatenate([[0], np.cumsum([p.size for p in parents])]).astype(np.int32)
    return offs, np.concatenate(parents), np.concatenate(probs)


@dataclasses.dataclass
class BudgetCase:
    """A batch-wide allocation workload: per-request candidate-tree specs
    (branching, depth_cap) or None, the batch capacity and the per-request
    node bound."""
    sizes: list
    capacity: int
    max_nodes: int


def budget_case(name):
    """Candidate batches shaped after the verification configs: each request
    drafts several times the nodes its share of the capacity can verify, and
    the capacity is the config's batch x tree size.
      tiny:       1 request, binary tree of depth 4 (31 candidates), capacity 15
      mid:        1 request, branching 4,4,2 to depth 8 (213), capacity 64
      production: 32 requests, branching 8,4,2 to depth 10 (553 each), capacity 2048
                  (32 x 64), max_nodes 128, so budgets vary between requests
      gdn:        16 requests, branching 16,4,2 to depth 8 (849 each), capacity 2048
                  (16 x 128), max_nodes 256
      large:      128 requests of mixed trees (branching 4,2,2 / 2,2,2 / 8,2 / a
                  chain of 16; 16-237 candidates), capacity 8192, max_nodes 256"""
    if name == "tiny":
        return BudgetCase([((2, 2, 2, 2), 4)], 15, 16)
    if name == "mid":
        return BudgetCase([((4, 4, 2), 8)], 64, 64)
    if name == "production":
        return BudgetCase([((8, 4, 2), 10)] * 32, 32 * 64, 128)
    if name == "gdn":
        return BudgetCase([((16, 4, 2), 8)] * 16, 16 * 128, 256)
    if name == "large":
        kinds = [((4, 2, 2), 16), ((2, 2, 2), 12), ((8, 2), 10), ((1,), 15)]
        return BudgetCase([kinds[b % 4] for b in range(128)], 8192, 256)
    raise KeyError(name)
