"""ctypes binding of libtreelin (argument marshalling only).

Every function takes torch tensors that already live on the GPU, passes their
device pointers and torch's current HIP stream to the C ABI declared in
include/treelin.h, and returns immediately (the work is asynchronous on that
stream).  A non-OK synchronous status raises TreeLinError.  The library must
have been built (python -m paper_2608_01651_amd.build); nothing here falls
back to another implementation.
"""
from __future__ import annotations

import ctypes
import os

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtreelin.so")

TL_OK, TL_EINVAL, TL_EBADTREE, TL_EBADPATH, TL_EUNSUPPORTED, TL_EHIP = range(6)
GLA, GDN = 0, 1
BF16, F32 = 0, 1


class TreeLinError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__(f"{where}: {status_string(status)}")


class Problem(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("num_qk_heads", ctypes.c_int32),
        ("num_v_heads", ctypes.c_int32),
        ("d_k", ctypes.c_int32),
        ("d_v", ctypes.c_int32),
        ("max_nodes", ctypes.c_int32),
        ("num_slots", ctypes.c_int32),
        ("mode", ctypes.c_int32),
        ("in_dtype", ctypes.c_int32),
        ("q_scale", ctypes.c_float),
    ]


class Layer(ctypes.Structure):
    """tl_layer: one layer's k, v, g, beta and state device pointers."""
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("g", ctypes.c_void_p),
                ("beta", ctypes.c_void_p), ("state", ctypes.c_void_p)]


MAX_COMMIT_LAYERS = 64
BUDGET_NOALLOC_MAX_BYTES = 1 << 20   # TL_BUDGET_NOALLOC_MAX_BYTES


def problem(batch, num_qk_heads, num_v_heads, d_k, d_v, max_nodes, num_slots=None,
            mode=GLA, in_dtype=BF16, q_scale=1.0):
    return Problem(batch, num_qk_heads, num_v_heads, d_k, d_v, max_nodes,
                   batch if num_slots is None else num_slots, mode, in_dtype, q_scale)


_lib = None


def lib():
    """The loaded shared library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with "
                               "`python -m paper_2608_01651_amd.build`")
        L = ctypes.CDLL(_LIB_PATH)
        P = ctypes.POINTER(Problem)
        vp = ctypes.c_void_p
        L.tree_lin_attn_verify.argtypes = [P] + [vp] * 12 + [ctypes.c_size_t, vp]
        L.tree_lin_attn_verify.restype = ctypes.c_int
        L.tree_state_commit.argtypes = [P] + [vp] * 12
        L.tree_state_commit.restype = ctypes.c_int
        L.tree_state_commit_layers.argtypes = [P, ctypes.c_int32, ctypes.POINTER(Layer)] + [vp] * 6
        L.tree_state_commit_layers.restype = ctypes.c_int
        L.tree_accepted_path.argtypes = [P] + [vp] * 7
        L.tree_accepted_path.restype = ctypes.c_int
        L.tree_conv_gates.argtypes = [P, ctypes.c_int32, ctypes.c_float] + [vp] * 18
        L.tree_conv_gates.restype = ctypes.c_int
        L.tree_conv_state_commit.argtypes = [P, ctypes.c_int32] + [vp] * 8
        L.tree_conv_state_commit.restype = ctypes.c_int
        L.tree_topology_export.argtypes = [P] + [vp] * 6
        L.tree_budget_select.argtypes = ([P, ctypes.c_int32, ctypes.c_int32] + [vp] * 9 +
                                         [ctypes.c_size_t, vp, vp])
        L.tree_budget_select.restype = ctypes.c_int
        L.tree_budget_select_noalloc.argtypes = [P, ctypes.c_int32, ctypes.c_int32] + [vp] * 10
        L.tree_budget_select_noalloc.restype = ctypes.c_int
        L.tree_budget_workspace_bytes.argtypes = [ctypes.c_int32, ctypes.c_int32]
        L.tree_budget_workspace_bytes.restype = ctypes.c_size_t
        L.tl_workspace_bytes.argtypes = [P]
        L.tl_workspace_bytes.restype = ctypes.c_size_t
        L.tree_topology_export.restype = ctypes.c_int
        L.tl_status_string.argtypes = [ctypes.c_int]
        L.tl_status_string.restype = ctypes.c_char_p
        L.tl_version.argtypes = []
        L.tl_version.restype = ctypes.c_char_p
        _lib = L
    return _lib


def status_string(status):
    return lib().tl_status_string(int(status)).decode()


def version():
    return lib().tl_version().decode()


_DT = {torch.int32: "int32", torch.float32: "float32", torch.bfloat16: "bfloat16",
       torch.int64: "int64"}


def _ptr(t, name, dtypes, optional=False):
    if t is None:
        if optional:
            return None
        raise ValueError(f"{name} is required")
    if isinstance(t, int):
        return t
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype not in dtypes:
        raise ValueError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr() or None


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


_IN = (torch.bfloat16, torch.float32)
_I32 = (torch.int32,)
_F32 = (torch.float32,)


def _check(status, where):
    if status != TL_OK:
        raise TreeLinError(status, where)


def workspace_bytes(prob):
    """tl_workspace_bytes: device workspace bytes verify needs for `prob`."""
    return int(lib().tl_workspace_bytes(ctypes.byref(prob)))


def verify(prob, node_offsets, parent, q, k, v, g, beta, state, out, slot=None,
           dev_err=None, workspace=None, stream=None):
    """tree_lin_attn_verify: writes out [N, Hv, d_v] fp32.  `workspace` is an
    optional uint8 device tensor of at least workspace_bytes(prob) bytes."""
    if workspace is None:
        ws_ptr, ws_bytes = None, 0
    else:
        if not isinstance(workspace, torch.Tensor) or not workspace.is_cuda or \
                workspace.dtype != torch.uint8:
            raise ValueError("workspace must be a uint8 CUDA (HIP) tensor")
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel()
    s = lib().tree_lin_attn_verify(
        ctypes.byref(prob), _ptr(node_offsets, "node_offsets", _I32), _ptr(parent, "parent", _I32),
        _ptr(q, "q", _IN), _ptr(k, "k", _IN), _ptr(v, "v", _IN), _ptr(g, "g", _F32),
        _ptr(beta, "beta", _F32, True), _ptr(state, "state", _F32), _ptr(slot, "slot", _I32, True),
        _ptr(out, "out", _F32), _ptr(dev_err, "dev_err", _I32, True), ws_ptr, ws_bytes,
        _stream(stream))
    _check(s, "tree_lin_attn_verify")


def commit(prob, node_offsets, parent, path_offsets, path, k, v, g, beta, state, slot=None,
           dev_err=None, stream=None):
    """tree_state_commit: overwrites the slots of requests with a non-empty path."""
    s = lib().tree_state_commit(
        ctypes.byref(prob), _ptr(node_offsets, "node_offsets", _I32), _ptr(parent, "parent", _I32),
        _ptr(path_offsets, "path_offsets", _I32), _ptr(path, "path", _I32, True),
        _ptr(k, "k", _IN), _ptr(v, "v", _IN), _ptr(g, "g", _F32), _ptr(beta, "beta", _F32, True),
        _ptr(state, "state", _F32), _ptr(slot, "slot", _I32, True),
        _ptr(dev_err, "dev_err", _I32, True), _stream(stream))
    _check(s, "tree_state_commit")


def topology(prob, node_offsets, parent, anc_mask, depth, dev_err=None, stream=None):
    """tree_topology_export: M+ rows [N, ceil(max_nodes/64)] (int64 bit patterns) and depths."""
    s = lib().tree_topology_export(
        ctypes.byref(prob), _ptr(node_offsets, "node_offsets", _I32), _ptr(parent, "parent", _I32),
        _ptr(anc_mask, "anc_mask", (torch.int64,)), _ptr(depth, "depth", _I32),
        _ptr(dev_err, "dev_err", _I32, True), _stream(stream))
    _check(s, "tree_topology_export")


def layer(k, v, g, beta, state):
    """One entry of commit_layers' layer table (checks dtypes and layout)."""
    return Layer(_ptr(k, "k", _IN), _ptr(v, "v", _IN), _ptr(g, "g", _F32),
                 _ptr(beta, "beta", _F32, True), _ptr(state, "state", _F32))


def commit_layers(prob, layers, node_offsets, parent, terminal, slot=None, dev_err=None,
                  stream=None):
    """tree_state_commit_layers: one launch commits every layer of `layers`
    (a list of layer(...) entries or of (k, v, g, beta, state) tuples) along
    the path that ends at terminal[b] (-1: nothing accepted)."""
    table = [x if isinstance(x, Layer) else layer(*x) for x in layers]
    arr = (Layer * max(1, len(table)))(*table)
    s = lib().tree_state_commit_layers(
        ctypes.byref(prob), len(table), arr, _ptr(node_offsets, "node_offsets", _I32),
        _ptr(parent, "parent", _I32), _ptr(terminal, "terminal", _I32),
        _ptr(slot, "slot", _I32, True), _ptr(dev_err, "dev_err", _I32, True), _stream(stream))
    _check(s, "tree_state_commit_layers")


def accepted_path(prob, node_offsets, parent, terminal, path_len, path, dev_err=None,
                  stream=None):
    """tree_accepted_path: path_len [B] and the root-first paths at path[node_offsets[b] + t]."""
    s = lib().tree_accepted_path(
        ctypes.byref(prob), _ptr(node_offsets, "node_offsets", _I32), _ptr(parent, "parent", _I32),
        _ptr(terminal, "terminal", _I32), _ptr(path_len, "path_len", _I32), _ptr(path, "path", _I32),
        _ptr(dev_err, "dev_err", _I32, True), _stream(stream))
    _check(s, "tree_accepted_path")


_BF = (torch.bfloat16,)


def conv_gates(prob, width, node_offsets, parent, x, gate_a, gate_b, conv_weight, conv_bias,
               A_log, dt_bias, conv_state, q, k, v, g, beta, slot=None, eps=1e-6, dev_err=None,
               stream=None):
    """tree_conv_gates: q, k, v (bf16) and g, beta (fp32) of every node from its
    mixed projection row x and its root-path convolution window."""
    s = lib().tree_conv_gates(
        ctypes.byref(prob), int(width), float(eps), _ptr(node_offsets, "node_offsets", _I32),
        _ptr(parent, "parent", _I32), _ptr(x, "x", _BF), _ptr(gate_a, "gate_a", _F32),
        _ptr(gate_b, "gate_b", _F32, True), _ptr(conv_weight, "conv_weight", _F32),
        _ptr(conv_bias, "conv_bias", _F32), _ptr(A_log, "A_log", _F32), _ptr(dt_bias, "dt_bias", _F32),
        _ptr(conv_state, "conv_state", _BF), _ptr(slot, "slot", _I32, True), _ptr(q, "q", _BF),
        _ptr(k, "k", _BF), _ptr(v, "v", _BF), _ptr(g, "g", _F32), _ptr(beta, "beta", _F32, True),
        _ptr(dev_err, "dev_err", _I32, True), _stream(stream))
    _check(s, "tree_conv_gates")


def conv_state_commit(prob, width, node_offsets, parent, terminal, x, conv_state, slot=None,
                      dev_err=None, stream=None):
    """tree_conv_state_commit: shifts the accepted path's x rows into the convolution state."""
    s = lib().tree_conv_state_commit(
        ctypes.byref(prob), int(width), _ptr(node_offsets, "node_offsets", _I32),
        _ptr(parent, "parent", _I32), _ptr(terminal, "terminal", _I32), _ptr(x, "x", _BF),
        _ptr(conv_state, "conv_state", _BF), _ptr(slot, "slot", _I32, True),
        _ptr(dev_err, "dev_err", _I32, True), _stream(stream))
    _check(s, "tree_conv_state_commit")


def budget_workspace_bytes(batch, max_nodes):
    """tree_budget_workspace_bytes: device bytes budget_select needs."""
    return int(lib().tree_budget_workspace_bytes(int(batch), int(max_nodes)))


def budget_workspace(batch, max_nodes, device="cuda"):
    """A workspace tensor for budget_select (uint8, 256-byte aligned by the allocator)."""
    return torch.empty(max(1, budget_workspace_bytes(batch, max_nodes)), dtype=torch.uint8, device=device)


def budget_select(prob, num_candidates, capacity, cand_offsets, cand_parent, cand_prob, rho, rank,
                  node_offsets, parent, src, workspace, dev_err=None, stream=None):
    """tree_budget_select: batch-wide allocation of `capacity` verification
    nodes over the candidate trees, packed into (node_offsets, parent, src)."""
    if not isinstance(workspace, torch.Tensor) or not workspace.is_cuda or workspace.dtype != torch.uint8:
        raise ValueError("workspace must be a uint8 CUDA (HIP) tensor")
    s = lib().tree_budget_select(
        ctypes.byref(prob), int(num_candidates), int(capacity),
        _ptr(cand_offsets, "cand_offsets", _I32), _ptr(cand_parent, "cand_parent", _I32),
        _ptr(cand_prob, "cand_prob", _F32), _ptr(rho, "rho", _F32), _ptr(rank, "rank", _I32),
        _ptr(node_offsets, "node_offsets", _I32), _ptr(parent, "parent", _I32),
        _ptr(src, "src", _I32), workspace.data_ptr(), workspace.numel(),
        _ptr(dev_err, "dev_err", _I32, True), _stream(stream))
    _check(s, "tree_budget_select")


def budget_select_noalloc(prob, num_candidates, capacity, cand_offsets, cand_parent, cand_prob,
                          rho, rank, node_offsets, parent, src, dev_err=None, stream=None):
    """tree_budget_select_noalloc: budget_select with the library's static
    per-GPU workspace (no allocation; calls overlapping on one GPU race)."""
    s = lib().tree_budget_select_noalloc(
        ctypes.byref(prob), int(num_candidates), int(capacity),
        _ptr(cand_offsets, "cand_offsets", _I32), _ptr(cand_parent, "cand_parent", _I32),
        _ptr(cand_prob, "cand_prob", _F32), _ptr(rho, "rho", _F32), _ptr(rank, "rank", _I32),
        _ptr(node_offsets, "node_offsets", _I32), _ptr(parent, "parent", _I32),
        _ptr(src, "src", _I32), _ptr(dev_err, "dev_err", _I32, True), _stream(stream))
    _check(s, "tree_budget_select_noalloc")
