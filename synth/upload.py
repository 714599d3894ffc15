"""Copy a synthetic workload to the GPU as contiguous torch tensors (plain
marshalling: int32 forest and paths, bf16 or fp32 q/k/v, fp32 gates)."""
from __future__ import annotations

import numpy as np
import torch


def _dev():
    return torch.device("cuda:0")


def t_int(x):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(x, dtype=np.int32))).to(_dev())


def t_f32(x):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(x, dtype=np.float32))).to(_dev())


def t_in(x, in_dtype):
    t = t_f32(x)
    return t if in_dtype == "f32" else t.to(torch.bfloat16)   # values are bf16-exact already


class Uploaded:
    def __init__(self, w):
        cfg = w.cfg
        self.w = w
        self.node_offsets = t_int(w.node_offsets)
        self.parent = t_int(w.parent) if w.N else torch.zeros(1, dtype=torch.int32, device=_dev())
        self.q = t_in(w.q, cfg.in_dtype)
        self.k = t_in(w.k, cfg.in_dtype)
        self.v = t_in(w.v, cfg.in_dtype)
        self.g = t_f32(w.g)
        self.beta = None if w.beta is None else t_f32(w.beta)
        self.path_offsets = t_int(w.path_offsets)
        self.path = t_int(w.path) if w.path.size else None
