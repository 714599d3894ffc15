"""Shared helpers for the GPU tests: upload a workload, build S_pre with the
oracle, run the library through its C ABI, and measure errors."""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2608_01651_amd import treelin as tl
from synth import workloads as W

TOL = 2e-3   # max relative error on outputs and committed states


from synth.upload import Uploaded, t_f32, t_in, t_int  # noqa: F401


def dev():
    return torch.device("cuda:0")


def oracle_prefix_state(cfg, seed, requests):
    """S_pre [len(requests), Hv, d_v, d_k] fp32: the oracle's recurrence over
    each request's synthetic prefix, from a zero state (fp64, rounded once)."""
    cfg = W.CONFIGS[cfg] if isinstance(cfg, str) else cfg
    out = []
    for b in requests:
        St = None
        for c in range(W.prefix_chunks(cfg)):
            k, v, g, beta = W.prefix_chunk(cfg, seed, b, c)
            grp = cfg.num_v_heads // cfg.num_qk_heads
            kh = k[:, np.arange(cfg.num_v_heads) // grp]
            St = oracle.prefix_state(cfg.mode, kh, v, g, beta, St0=St)
        out.append(St)
    return np.stack(out).astype(np.float32)


def problem_for(cfg, batch, num_slots=None):
    return tl.problem(batch, cfg.num_qk_heads, cfg.num_v_heads, cfg.d_k, cfg.d_v, cfg.max_nodes,
                      num_slots=num_slots, mode=cfg.mode,
                      in_dtype=tl.F32 if cfg.in_dtype == "f32" else tl.BF16, q_scale=cfg.q_scale)


def run_verify(cfg, up: Uploaded, state_t, slot=None, num_slots=None, max_nodes=None):
    prob = problem_for(cfg, up.w.batch, num_slots=num_slots if num_slots else state_t.shape[0])
    if max_nodes:
        prob.max_nodes = max_nodes
    out = torch.full((max(up.w.N, 1), cfg.num_v_heads, cfg.d_v), float("nan"), device=dev())
    err = torch.zeros(1, dtype=torch.int32, device=dev())
    tl.verify(prob, up.node_offsets, up.parent, up.q, up.k, up.v, up.g, up.beta, state_t, out,
              slot=slot, dev_err=err)
    torch.cuda.synchronize()
    return out[:up.w.N].cpu().numpy(), int(err.item())


def run_commit(cfg, up: Uploaded, state_t, slot=None, num_slots=None):
    prob = problem_for(cfg, up.w.batch, num_slots=num_slots if num_slots else state_t.shape[0])
    err = torch.zeros(1, dtype=torch.int32, device=dev())
    tl.commit(prob, up.node_offsets, up.parent, up.path_offsets, up.path, up.k, up.v, up.g,
              up.beta, state_t, slot=slot, dev_err=err)
    torch.cuda.synchronize()
    return int(err.item())


def slice_rel_err(got, ref, node_offsets):
    """Worst over (request, v-head) of max|got - ref| / max|ref| on that
    request's [T_b, d_v] output slice."""
    worst = 0.0
    for b in range(len(node_offsets) - 1):
        o0, o1 = int(node_offsets[b]), int(node_offsets[b + 1])
        if o1 == o0:
            continue
        d = np.abs(got[o0:o1].astype(np.float64) - ref[o0:o1])     # [T, Hv, dv]
        scale = np.abs(ref[o0:o1]).max(axis=(0, 2))
        err = d.max(axis=(0, 2))
        for h in range(d.shape[1]):
            e = err[h] / scale[h] if scale[h] > 0 else (err[h] if err[h] > 1e-6 else 0.0)
            worst = max(worst, float(e))
    return worst


def state_rel_err(got, ref):
    """Worst over (slot, head) of max|got - ref| / max|ref| on the [d_v, d_k] state."""
    d = np.abs(got.astype(np.float64) - ref).max(axis=(2, 3))
    s = np.abs(ref).max(axis=(2, 3))
    e = np.where(s > 0, d / np.where(s > 0, s, 1), np.where(d > 1e-6, d, 0))
    return float(e.max()) if e.size else 0.0
