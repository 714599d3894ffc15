"""Validity of a budget selection that does not depend on the precision of rho
(§5.1 "Batch-wide utility allocation").

The allocation keeps every root, then takes the batch's highest-rho
candidates (at most max_nodes nodes per request) until the capacity is
spent, and packs them per request in candidate order.  Where exact rho values
lie within rounding of the cut, several selections are correct; the bit-exact
parity tests accept only the one the fp32 arithmetic picks.  This check
accepts every selection that is correct for SOME rho within the fp32
rounding bound of the exact one:

* rho is recomputed here in fp64 from the parents and probabilities (the
  probabilities are fp32 inputs, exact in fp64); a step-wise fp32 product of
  k + 1 factors is within (k + 1) u (u = 2^-24) relative of it, plus one
  subnormal spacing per step where it underflows;
* the packed forest is well formed: budgets sum to min(capacity, the most
  the caps allow), each request keeps all its roots and at most max_nodes
  nodes, in candidate order, with packed parents naming the candidate's own
  parent (so the kept set is prefix-connected);
* the cut: every candidate left out of a request that is not full scores,
  up to the bound, no higher than every selected non-root in the batch; in
  a full request, no higher than every selected non-root of that request.
"""
from __future__ import annotations

import numpy as np

U32 = 2.0 ** -24      # unit roundoff of fp32
TINY = 2.0 ** -149    # spacing of fp32 subnormals


def rho_fp64(offs, parent, prob):
    """Exact-ish rho (fp64 product along the root path) and node depths."""
    M = int(offs[-1])
    rho = np.zeros(M)
    depth = np.zeros(M, np.int64)
    for b in range(len(offs) - 1):
        o0, o1 = int(offs[b]), int(offs[b + 1])
        for v in range(o1 - o0):
            p = int(parent[o0 + v])
            if p == -1:
                rho[o0 + v] = float(prob[o0 + v])
            else:
                rho[o0 + v] = rho[o0 + p] * float(prob[o0 + v])
                depth[o0 + v] = depth[o0 + p] + 1
    return rho, depth


def check_selection(offs, parent, prob, capacity, max_nodes, node_offsets, fparent, src):
    """Assert that (node_offsets, fparent, src) is a correct allocation of the
    candidate batch (offs, parent, prob) for some rho within the fp32 bound."""
    offs = np.asarray(offs, np.int64)
    parent = np.asarray(parent, np.int64)
    node_offsets = np.asarray(node_offsets, np.int64)
    B, M = len(offs) - 1, int(offs[-1])
    rho, depth = rho_fp64(offs, parent, prob)
    err = (depth + 1) * U32 * 1.001 * rho + (depth + 1) * TINY
    hi, lo = rho + err, rho - err          # bounds of what the fp32 rho can be

    assert node_offsets.shape == (B + 1,) and node_offsets[0] == 0
    assert np.all(np.diff(node_offsets) >= 0)
    N = int(node_offsets[-1])
    sizes = np.diff(offs)
    assert N == min(capacity, int(np.minimum(sizes, max_nodes).sum())), "budgets do not fill the capacity"
    src = np.asarray(src, np.int64)[:N]
    fparent = np.asarray(fparent, np.int64)[:N]
    chosen = np.zeros(M, bool)
    full = np.zeros(B, bool)
    for b in range(B):
        n0, n1 = int(node_offsets[b]), int(node_offsets[b + 1])
        o0, o1 = int(offs[b]), int(offs[b + 1])
        s, p = src[n0:n1], fparent[n0:n1]
        assert n1 - n0 <= max_nodes, f"request {b} exceeds max_nodes"
        assert np.all((s >= o0) & (s < o1)), f"request {b} takes another request's candidates"
        assert np.all(np.diff(s) > 0), f"request {b} is not in candidate order"
        for i in range(n1 - n0):
            cp = int(parent[s[i]])
            if cp == -1:
                assert p[i] == -1, f"request {b}: root {s[i]} given a parent"
            else:
                assert 0 <= p[i] < i and s[p[i]] - o0 == cp, f"request {b}: parent link of {s[i]}"
        chosen[s] = True
        roots = np.flatnonzero(parent[o0:o1] == -1) + o0
        assert chosen[roots].all(), f"request {b} drops a root"
        full[b] = (n1 - n0) == max_nodes
    req = np.repeat(np.arange(B), sizes)
    sel = chosen & (parent != -1)
    out = ~chosen
    if sel.any() and (out & ~full[req]).any():
        worst_in = hi[sel].min()
        best_out = lo[out & ~full[req]].max()
        assert best_out <= worst_in, f"left out rho {best_out} above selected {worst_in}"
    for b in np.flatnonzero(full):
        m = req == b
        if (sel & m).any() and (out & m).any():
            assert lo[out & m].max() <= hi[sel & m].min(), f"full request {b}: cut out of order"
