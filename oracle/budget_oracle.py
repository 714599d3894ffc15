"""Oracle for the batch-wide verification-budget allocation and the forest
materialiser (§5.1 "Batch-wide utility allocation", §5.2 "CUDA
Graph-native packed-forest execution").

TEST INFRASTRUCTURE ONLY, like tree_oracle: only the tests, the smoke check
and the benchmark's CPU-baseline leg may import it, and it shares no code
with the HIP path.

What is computed
----------------
* Each request brings a candidate tree (parents before children, -1 for a
  root) with the drafter's probability p(u | parent(u)) per node.  A node's
  utility is rho(v) = prod_{u in P(v)} p(u | parent(u)), P(v) its root path.
* Every root of a request with candidates is kept.  The remaining capacity
  is filled with the highest-rho candidates across the whole batch.  A
  child's rho never exceeds its parent's, so each request's selection is
  prefix-connected.
* A segmented count gives each request's budget; the selected nodes are
  packed, request by request and in candidate order (a topological order),
  into the flat forest: node_offsets, parents in packed numbering, and the
  candidate row of every packed node.

Readings (the paper leaves these open; the kernels take the same ones)
-------------------------------------------------------------------
* rho is formed in fp32, root first, one rounding per step:
  rho(root) = p(root), rho(v) = fl32(rho(parent) * p(v)).  Its bits decide
  the selection, so the oracle takes that decision in the kernel's precision.
* Order: larger rho first; equal rho, lower batch-wide candidate index first
  (so a parent always precedes its children).
* Each request keeps at most max_nodes nodes (the verification kernels'
  bound): a candidate is eligible only while it ranks below
  max_nodes - (roots of its request) among its request's non-root
  candidates, i.e. the greedy selection skips a request once it is full.
* The capacity must cover every root of every request with candidates.
* Draft probabilities lie in [0, 1]: that bound is what keeps a child's rho
  at or below its parent's, so a value outside it (or NaN) is rejected.
"""
from __future__ import annotations

import numpy as np

from .tree_oracle import BadTree, InvalidArg


def path_scores(cand_parent, cand_prob):
    """rho of one request's candidates, fp32, root first."""
    T = len(cand_parent)
    rho = np.zeros(T, dtype=np.float32)
    for v in range(T):
        p = int(cand_parent[v])
        if not (p == -1 or 0 <= p < v):
            raise BadTree(f"candidate {v}: parent {p} is not -1 or in [0,{v})")
        if not (0.0 <= float(cand_prob[v]) <= 1.0):
            raise InvalidArg(f"candidate {v}: probability {cand_prob[v]} is outside [0, 1]")
        rho[v] = cand_prob[v] if p == -1 else np.float32(rho[p] * np.float32(cand_prob[v]))
    return rho


def order_key(rho, v):
    """Selection order: larger rho first, then the lower batch-wide index."""
    return (-float(rho[v]), v)


def room(max_nodes, roots):
    """Non-root nodes a request may keep."""
    return max_nodes - roots


def budget_select(cand_offsets, cand_parent, cand_prob, capacity, max_nodes):
    """Returns dict(rho [M] fp32, rank [M] int32 (-1 for roots), node_offsets
    [B+1], parent [N] packed, src [N] candidate rows)."""
    cand_offsets = np.asarray(cand_offsets, np.int64)
    cand_prob = np.asarray(cand_prob, np.float32)
    B = cand_offsets.size - 1
    M = int(cand_offsets[-1])
    rho = np.zeros(M, np.float32)
    rank = np.full(M, -1, np.int32)
    roots = np.zeros(B, np.int64)
    for b in range(B):
        o0, o1 = int(cand_offsets[b]), int(cand_offsets[b + 1])
        if o1 < o0:
            raise BadTree("cand_offsets must be non-decreasing")
        par = np.asarray(cand_parent[o0:o1])
        rho[o0:o1] = path_scores(par, cand_prob[o0:o1])
        roots[b] = int((par == -1).sum())
        if roots[b] > max_nodes:
            raise InvalidArg(f"request {b} has more roots than max_nodes")
        # rank of every non-root candidate within its request
        nonroot = [v for v in range(o0, o1) if cand_parent[v] != -1]
        nonroot.sort(key=lambda v: order_key(rho, v))
        for r, v in enumerate(nonroot):
            rank[v] = r
    if capacity < roots.sum():
        raise InvalidArg("capacity is below the number of roots")
    # the global selection over eligible candidates
    req = np.repeat(np.arange(B), np.diff(cand_offsets))
    eligible = [v for v in range(M) if rank[v] >= 0 and rank[v] < room(max_nodes, roots[req[v]])]
    eligible.sort(key=lambda v: order_key(rho, v))
    chosen = set(eligible[:max(0, int(capacity - roots.sum()))])
    selected = [v for v in range(M) if rank[v] < 0 or v in chosen]
    # segmented counts and packing
    counts = np.zeros(B, np.int64)
    for v in selected:
        counts[req[v]] += 1
    node_offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    parent = np.zeros(len(selected), np.int32)
    src = np.zeros(len(selected), np.int32)
    packed = {}
    for b in range(B):
        k = int(node_offsets[b])
        for v in range(int(cand_offsets[b]), int(cand_offsets[b + 1])):
            if rank[v] < 0 or v in chosen:
                local = k - int(node_offsets[b])
                packed[v] = local
                p = int(cand_parent[v])
                if p != -1 and (int(cand_offsets[b]) + p) not in packed:
                    raise AssertionError("selection is not prefix-connected")
                parent[k] = -1 if p == -1 else packed[int(cand_offsets[b]) + p]
                src[k] = v
                k += 1
    return dict(rho=rho, rank=rank, node_offsets=node_offsets, parent=parent, src=src)
