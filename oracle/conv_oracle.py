"""fp64 CPU oracle for the tree-parallel front end of a gated linear-attention
layer: the short causal depthwise convolution, bias, SiLU, q/k normalisation
and gate preparation over a drafted token tree, and the commit of the
convolution state along the accepted path.

TEST INFRASTRUCTURE ONLY, like tree_oracle: only the tests, the smoke check
and the benchmark's CPU-baseline leg may import it, and it shares no code
with the HIP path.

What is computed, and where the paper defines it
------------------------------------------------
* §2.1: a GDN layer forms its recurrent operands with a short causal
  depthwise convolution and input-dependent gates.
* §4.3, Stage 1: on a sequence the convolution reads a fixed number of
  preceding tokens; for a tree node those tokens lie on its root-to-node
  path, so each node follows parent links.  Convolution, bias, SiLU and gate
  preparation are fused per node.
* Near the root the window reaches back into the committed prefix: the
  request's convolution state holds the last width-1 inputs of the prefix
  (the sequential rule applied to the prefix, restated for the tree).
* The commit keeps, as the new convolution state, the last width-1 inputs of
  the sequence prefix + accepted path (the accepted path of §4.4).

Readings (the paper fixes none of these formulas; the kernels take the same ones)
------------------------------------------------------------------------------
* x[r] is the node's mixed projection row [q | k | v] of
  C = 2 Hk d_k + Hv d_v channels.  Channel c of node i:
    y_i[c] = bias[c] + sum_{p=0}^{w-1} W[c, p] * s_i[p][c],
  where s_i is the last w rows of (conv_state rows, x rows of Anc(i) u {i}
  root first); p = w-1 is the node itself.  z = SiLU(y) = y sigmoid(y).
* q and k are normalised per head: z / sqrt(sum z^2 + eps).
* Gates of the Gated DeltaNet parameterisation: per (node, v-head)
    g    = -exp(A_log[h]) * softplus(a[i, h] + dt_bias[h])   (log-decay)
    beta = sigmoid(b[i, h])                                   (delta rule only)
"""
from __future__ import annotations

import numpy as np

from .tree_oracle import (BadPath, BadTree, GDN, GLA, InvalidArg, MAX_NODES_LIMIT,
                          check_forest, root_path)


def _softplus(x):
    return np.logaddexp(0.0, x)


def _sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


def _slot_of(slot, b):
    return b if slot is None else int(slot[b])


def channels(num_qk_heads, num_v_heads, d_k, d_v):
    return 2 * num_qk_heads * d_k + num_v_heads * d_v


def conv_window(conv_state_b, x_rows_root_first, width):
    """The last `width` rows of (committed state rows, path rows): the
    convolution window of the path's last node, oldest row first."""
    seq = np.concatenate([conv_state_b, x_rows_root_first], axis=0)
    return seq[-width:]


def conv_gates(mode, num_qk_heads, num_v_heads, d_k, d_v, width, node_offsets, parent,
               x, gate_a, gate_b, conv_weight, conv_bias, A_log, dt_bias, conv_state,
               slot=None, eps=1e-6, max_nodes=MAX_NODES_LIMIT):
    """q [N, Hk, d_k], k [N, Hk, d_k], v [N, Hv, d_v], g [N, Hv], beta [N, Hv]
    (None for gated linear attention), all float64."""
    if mode not in (GLA, GDN):
        raise InvalidArg("unknown mode")
    if (mode == GDN) != (gate_b is not None):
        raise InvalidArg("gate_b is needed by, and only by, the delta rule")
    if not (2 <= width <= 4):
        raise InvalidArg("conv width must lie in [2, 4]")
    check_forest(node_offsets, parent, max_nodes)
    Hk, Hv = num_qk_heads, num_v_heads
    C = channels(Hk, Hv, d_k, d_v)
    x = np.asarray(x, np.float64)
    N = x.shape[0]
    if x.shape != (N, C) or conv_weight.shape != (C, width) or conv_bias.shape != (C,):
        raise InvalidArg("x must be [N, C], conv_weight [C, width], conv_bias [C]")
    cs = np.asarray(conv_state, np.float64)
    if cs.ndim != 3 or cs.shape[1:] != (width - 1, C):
        raise InvalidArg("conv_state must be [slots, width - 1, C]")
    W = np.asarray(conv_weight, np.float64)
    bias = np.asarray(conv_bias, np.float64)
    z = np.zeros((N, C))
    for b in range(len(node_offsets) - 1):
        o = int(node_offsets[b])
        pb = np.asarray(parent[o:int(node_offsets[b + 1])])
        for i in range(pb.size):
            rows = x[[o + t for t in root_path(pb, i)]]
            win = conv_window(cs[_slot_of(slot, b)], rows, width)      # [width, C]
            y = bias + np.einsum("cp,pc->c", W, win)
            z[o + i] = y * _sigmoid(y)
    nq = Hk * d_k
    q = z[:, :nq].reshape(N, Hk, d_k)
    k = z[:, nq:2 * nq].reshape(N, Hk, d_k)
    v = z[:, 2 * nq:].reshape(N, Hv, d_v)
    q = q / np.sqrt((q * q).sum(-1, keepdims=True) + eps)
    k = k / np.sqrt((k * k).sum(-1, keepdims=True) + eps)
    a = np.asarray(gate_a, np.float64)
    g = -np.exp(np.asarray(A_log, np.float64))[None, :] * _softplus(a + np.asarray(dt_bias, np.float64)[None, :])
    beta = None if gate_b is None else _sigmoid(np.asarray(gate_b, np.float64))
    return q, k, v, g, beta


def conv_state_commit(width, node_offsets, parent, terminal, x, conv_state, slot=None,
                      max_nodes=MAX_NODES_LIMIT):
    """New convolution states: for request b with terminal node a, the last
    width-1 rows of (its committed state rows, x rows of Anc(a) u {a} root
    first); terminal -1 keeps the slot.  Returns a new array; slots no
    request names are copied through."""
    check_forest(node_offsets, parent, max_nodes)
    cs = np.array(conv_state, np.float64)
    new = cs.copy()
    x = np.asarray(x, np.float64)
    for b in range(len(node_offsets) - 1):
        o, T = int(node_offsets[b]), int(node_offsets[b + 1] - node_offsets[b])
        a = int(terminal[b])
        if not (-1 <= a < T):
            raise BadPath(f"request {b}: terminal {a} outside [-1,{T})")
        if a == -1:
            continue
        rows = x[[o + t for t in root_path(np.asarray(parent[o:o + T]), a)]]
        s = _slot_of(slot, b)
        new[s] = np.concatenate([cs[s], rows], axis=0)[-(width - 1):]
    return new


__all__ = ["channels", "conv_window", "conv_gates", "conv_state_commit", "BadTree", "BadPath"]
