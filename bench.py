"""Benchmark: verified tree-tokens/s per linear-attention layer on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload production]

One step is one pass of the hot path over one batch: tree-parallel verify of
one layer's draft forest, then the accepted-path commit of that layer's state.
The timed loop keeps R independent layer buffer sets resident in HBM (R chosen
so the sets exceed twice the 256 MB Infinity Cache) and runs, per round,
verify over all R layers and then commit over the same R layers -- the order
of a real forward pass, where every layer verifies before sampling and the
commit follows.  Inputs are resident before timing starts; the step count is
rounded up to a multiple of R.

The JSON line reports whole-job throughput (tree tokens / s per layer), the
HIP-event average duration of each kernel, the algorithmic HBM bytes each
kernel must move, the roofline of the dominant kernel against the MI355X's
8 TB/s, and the fp64 oracle timed on host cores over a bounded sample.
"""
from __future__ import annotations

import argparse
import dataclasses
import re
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MALL_BYTES = 256 << 20
METRIC = "verified tree-tokens/s per linear-attn layer; % of HBM roofline (1 MI355X)"


# ---------------------------------------------------------------------------
# algorithmic bytes (what the method must move; no per-node state traffic)
# ---------------------------------------------------------------------------
def verify_bytes(cfg, N, B):
    Q = 4 if cfg.in_dtype == "f32" else 2
    gdn = 1 if cfg.mode == 1 else 0
    Hk, Hv, dk, dv = cfg.num_qk_heads, cfg.num_v_heads, cfg.d_k, cfg.d_v
    per_node = 2 * Hk * dk * Q + Hv * dv * Q + Hv * 4 * (1 + gdn) + 4
    return N * per_node + 4 * (B + 1) + B * Hv * dk * dv * 4 + N * Hv * dv * 4


def commit_bytes(cfg, path_lens):
    Q = 4 if cfg.in_dtype == "f32" else 2
    gdn = 1 if cfg.mode == 1 else 0
    Hk, Hv, dk, dv = cfg.num_qk_heads, cfg.num_v_heads, cfg.d_k, cfg.d_v
    L = np.asarray(path_lens)
    per_row = Hk * dk * Q + Hv * dv * Q + Hv * 4 * (1 + gdn) + 4
    return int((L > 0).sum()) * 2 * Hv * dk * dv * 4 + int(L.sum()) * per_row + 4 * (L.size + 1)


def conv_bytes(cfg, N, B, width):
    """tree_conv_gates: every node's mixed row read once and q/k/v written
    once (bf16), the gate inputs and outputs, the requests' state rows, the
    layer's parameters and the forest.  A node's ancestor rows are the
    ancestors' own rows: they are not counted again."""
    gdn = 1 if cfg.mode == 1 else 0
    Hk, Hv, dk, dv = cfg.num_qk_heads, cfg.num_v_heads, cfg.d_k, cfg.d_v
    C = 2 * Hk * dk + Hv * dv
    per_node = 2 * C * 2 + 2 * Hv * 4 * (1 + gdn) + 4
    return N * per_node + B * (width - 1) * C * 2 + C * (width + 1) * 4 + 2 * Hv * 4 + 4 * (B + 1)


# The sources that the verify and commit launches of the benchmark compile from.
HASHED_SOURCES = ["include/treelin.h"] + [
    "paper_2608_01651_amd/csrc/" + f for f in
    ("tl_device.h", "tl_kernels.h", "verify_common.h", "verify_gdn.h", "verify_gla_small.h",
     "verify_vector.h", "verify.hip", "verify_tiled.hip", "verify_gla_large.hip", "verify_gdn_dense.hip",
     "commit.hip")]


def source_hash():
    """Hash of the verify and commit kernels' source code: comments and
    whitespace are dropped, so that only a change to what those kernels
    compile from invalidates stored counters."""
    h = hashlib.sha256()
    for f in HASHED_SOURCES:
        with open(os.path.join(ROOT, f), encoding="utf-8") as fh:
            code = re.sub(r"/\*.*?\*/", " ", fh.read(), flags=re.S)
        code = re.sub(r"//[^\n]*", " ", code)
        h.update(os.path.basename(f).encode() + " ".join(code.split()).encode())
    return h.hexdigest()[:16]


# ---------------------------------------------------------------------------
# GPU leg
# ---------------------------------------------------------------------------
class LayerSet:
    """One layer's resident inputs: the forest, q/k/v/gates and its state slots."""

    def __init__(self, w, state_t, torch):
        from synth.upload import Uploaded
        self.up = Uploaded(w)
        self.state = state_t
        self.out = torch.empty((w.N, w.cfg.num_v_heads, w.cfg.d_v), dtype=torch.float32,
                               device=state_t.device)


def build_prefix_state_gpu(cfg, seed, batch, torch, tl, log):
    """S_pre of every request: the library's own commit replays each request's
    synthetic prefix (chunks of 256 tokens as chain trees) from a zero state."""
    from synth import workloads as W
    dev = torch.device("cuda:0")
    state = torch.zeros((batch, cfg.num_v_heads, cfg.d_v, cfg.d_k), dtype=torch.float32, device=dev)
    prob = tl.problem(batch, cfg.num_qk_heads, cfg.num_v_heads, cfg.d_k, cfg.d_v, W.PREFIX_CHUNK,
                      mode=cfg.mode, in_dtype=tl.F32 if cfg.in_dtype == "f32" else tl.BF16)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    in_t = torch.float32 if cfg.in_dtype == "f32" else torch.bfloat16
    for c in range(W.prefix_chunks(cfg)):
        parts = [W.prefix_chunk(cfg, seed, b, c) for b in range(batch)]
        L = parts[0][0].shape[0]
        offs = torch.arange(0, (batch + 1) * L, L, dtype=torch.int32, device=dev)
        parent = torch.arange(-1, L - 1, dtype=torch.int32, device=dev).repeat(batch)
        path = torch.arange(0, L, dtype=torch.int32, device=dev).repeat(batch)
        k = torch.from_numpy(np.concatenate([p[0] for p in parts])).to(dev).to(in_t)
        v = torch.from_numpy(np.concatenate([p[1] for p in parts])).to(dev).to(in_t)
        g = torch.from_numpy(np.concatenate([p[2] for p in parts])).to(dev)
        beta = None if parts[0][3] is None else torch.from_numpy(np.concatenate([p[3] for p in parts])).to(dev)
        tl.commit(prob, offs, parent, offs, path, k, v, g, beta, state, dev_err=err)
    torch.cuda.synchronize()
    if err.item() != 0:
        raise RuntimeError(f"prefix commit reported {tl.status_string(err.item())}")
    log(f"prefix state built from {cfg.prefix_len} tokens per request")
    return state


def sample_requests(cfg):
    """Requests the oracle checks in each run: the first, the second (in the
    large workload request 0 is the 16-node chain and request 1 the 256-node
    tree), the middle and the last."""
    B = cfg.batch
    return sorted({0, min(1, B - 1), B // 2, B - 1})


def slice_rel_err(got, ref, node_offsets):
    """Worst over (request, v-head) of max|got - ref| / max|ref| over that
    request's [T_b, d_v] output slice (the normwise error the tolerance is
    stated in)."""
    worst = 0.0
    for b in range(len(node_offsets) - 1):
        o0, o1 = int(node_offsets[b]), int(node_offsets[b + 1])
        if o1 == o0:
            continue
        d = np.abs(got[o0:o1].astype(np.float64) - ref[o0:o1]).max(axis=(0, 2))
        scale = np.abs(ref[o0:o1]).max(axis=(0, 2))
        for h in range(d.size):
            e = d[h] / scale[h] if scale[h] > 0 else (d[h] if d[h] > 1e-6 else 0.0)
            worst = max(worst, float(e))
    return worst


def state_rel_err(got, ref):
    """Worst over (slot, v-head) of max|got - ref| / max|ref| over the [d_v, d_k] state."""
    d = np.abs(got.astype(np.float64) - ref).max(axis=(-2, -1))
    sc = np.abs(ref).max(axis=(-2, -1))
    e = np.where(sc > 0, d / np.where(sc > 0, sc, 1), np.where(d > 1e-6, d, 0))
    return float(e.max()) if e.size else 0.0


def gpu_leg(args, cfg, log, check=None, steps=None, warmup=None):
    """Times the hot path on one workload.  `check` (from the CPU leg) holds
    the oracle's S_pre, outputs and committed states of sampled requests;
    their slots start from that S_pre and one untimed step, launched exactly
    as the timed ones, is compared with it."""
    import torch
    from paper_2608_01651_amd import treelin as tl
    from synth import workloads as W

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU (HIP) device")
    tl.lib()   # fail loudly if the library is missing
    steps = args.steps if steps is None else steps
    warmup = args.warmup if warmup is None else warmup
    w = W.make(cfg, seed=args.seed)
    log(f"workload {cfg.name}: B={w.batch} N={w.N} paths={int(w.path.size)} rows")
    if cfg.prefix_len:
        state0 = build_prefix_state_gpu(cfg, args.seed, w.batch, torch, tl, log)
    else:
        state0 = torch.from_numpy(w.state).to("cuda:0")
    if check is not None:
        idx = torch.tensor(check["sample"], dtype=torch.long, device="cuda:0")
        state0[idx] = torch.from_numpy(check["state_pre"]).to("cuda:0")
    vb = verify_bytes(cfg, w.N, w.batch)
    cb = commit_bytes(cfg, np.diff(w.path_offsets))
    # a layer set's footprint is what verify touches: state, q/k/v/gates,
    # output; enough sets to exceed the Infinity Cache twice, at most 64 (the
    # latency-bound shapes have footprints of kilobytes, and a captured round
    # holds two launches per set)
    R = args.layers or min(64, max(1, math.ceil(2 * MALL_BYTES / vb)))
    sets = []
    for r in range(R):
        sets.append(LayerSet(w, state0.clone(), torch))
    log(f"{R} layer sets resident ({R * vb / 1e6:.0f} MB of verify footprint)")
    prob = tl.problem(w.batch, cfg.num_qk_heads, cfg.num_v_heads, cfg.d_k, cfg.d_v, cfg.max_nodes,
                      mode=cfg.mode, in_dtype=tl.F32 if cfg.in_dtype == "f32" else tl.BF16,
                      q_scale=cfg.q_scale)
    err = torch.zeros(1, dtype=torch.int32, device="cuda:0")
    stream = torch.cuda.current_stream()

    def run_verify(s):
        u = s.up
        tl.verify(prob, u.node_offsets, u.parent, u.q, u.k, u.v, u.g, u.beta, s.state, s.out,
                  dev_err=err)

    def run_commit(s):
        u = s.up
        tl.commit(prob, u.node_offsets, u.parent, u.path_offsets, u.path, u.k, u.v, u.g, u.beta,
                  s.state, dev_err=err)

    # the unified commit: every layer set in one call, each request's path
    # given by its terminal node
    terminal = torch.tensor([int(w.path[w.path_offsets[b + 1] - 1]) if w.path_offsets[b + 1] > w.path_offsets[b]
                             else -1 for b in range(w.batch)], dtype=torch.int32, device="cuda:0")
    table = [tl.layer(s.up.k, s.up.v, s.up.g, s.up.beta, s.state) for s in sets]

    def run_commits():
        if args.commit_layers:
            tl.commit_layers(prob, table, sets[0].up.node_offsets, sets[0].up.parent, terminal,
                             dev_err=err)
        else:
            for s in sets:
                run_commit(s)

    checked = None
    if check is not None:
        # one step of layer set 0, launched as in the timed loop, against the
        # oracle on the sampled requests; then the set's state is restored
        run_verify(sets[0])
        run_commits()
        torch.cuda.synchronize()
        if err.item() != 0:
            raise RuntimeError(f"device error {tl.status_string(err.item())}")
        sample = check["sample"]
        rows = np.concatenate([np.arange(w.node_offsets[b], w.node_offsets[b + 1]) for b in sample])
        got_o = sets[0].out.cpu().numpy()[rows]
        got_s = sets[0].state.cpu().numpy()[sample]
        sub_offs = np.concatenate([[0], np.cumsum(np.diff(w.node_offsets)[sample])])
        e_o = slice_rel_err(got_o, check["ref_out"], sub_offs)
        e_s = state_rel_err(got_s, check["ref_state"])
        finite = bool(np.isfinite(sets[0].out.cpu().numpy()).all() and
                      torch.isfinite(sets[0].state).all().item())
        checked = {"max_rel_err_out": float(f"{e_o:.3e}"), "max_rel_err_state": float(f"{e_s:.3e}"),
                   "tolerance": 2e-3, "pass": bool(e_o <= 2e-3 and e_s <= 2e-3 and finite),
                   "all_outputs_finite": finite, "requests": [int(b) for b in sample],
                   "what": "one untimed step (verify + commit of layer set 0, the timed loop's launches) "
                           "against the fp64 oracle on the sampled requests, whose S_pre is the oracle's "
                           "prefix recurrence; normwise max relative error per (request, v-head)"}
        log(f"oracle check on requests {sample}: out {e_o:.2e}, state {e_s:.2e}")
        for s in sets:
            s.state.copy_(state0)
        torch.cuda.synchronize()

    rounds_w = max(1, math.ceil(warmup / R))
    for _ in range(rounds_w):
        for s in sets:
            run_verify(s)
        run_commits()
    torch.cuda.synchronize()
    if err.item() != 0:
        raise RuntimeError(f"device error {tl.status_string(err.item())}")

    rounds = max(1, math.ceil(steps / R))
    nsteps = rounds * R

    def one_round():
        for s in sets:
            run_verify(s)
        run_commits()

    graph = None
    if args.graph:
        # one round (R verifies, then the commits) captured once and replayed;
        # the kernels read every size from device memory, so replays need no
        # host work
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            one_round()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            one_round()
        torch.cuda.synchronize()
        for _ in range(rounds_w):
            graph.replay()
        torch.cuda.synchronize()

    def timed(body):
        # only a start and an end event around the launches, on the stream
        # they are enqueued on (markers between kernels would perturb them)
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record(stream)
        for _ in range(rounds):
            body()
        end.record(stream)
        torch.cuda.synchronize()
        return start.elapsed_time(end)

    def verify_only():
        for s in sets:
            run_verify(s)

    t_host0 = time.perf_counter()
    total_ms = timed(graph.replay if graph is not None else one_round)
    wall = time.perf_counter() - t_host0
    if err.item() != 0:
        raise RuntimeError(f"device error {tl.status_string(err.item())}")
    # each kernel alone: its launches back to back over the same layer sets,
    # as many as in the timed steps (the per-kernel average launch duration)
    v_ms = timed(verify_only) / (rounds * R)
    c_ms = timed(run_commits) / (rounds * R)
    if err.item() != 0:
        raise RuntimeError(f"device error {tl.status_string(err.item())}")
    log(f"timed {nsteps} steps: {total_ms:.3f} ms (host wall {wall * 1e3:.1f} ms); "
        f"kernel passes: verify {v_ms * 1e3:.2f} us, commit {c_ms * 1e3:.2f} us per launch")
    return dict(w=w, steps=nsteps, R=R, total_ms=total_ms, verify_ms=v_ms, commit_ms=c_ms,
                verify_bytes=vb, commit_bytes=cb, check=checked)


def conv_leg(args, cfg, log):
    """Times tree_conv_gates over resident layer sets (bf16 inputs)."""
    import torch
    from paper_2608_01651_amd import treelin as tl
    from synth import workloads as W

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU (HIP) device")
    tl.lib()
    cfg = dataclasses.replace(cfg, in_dtype="bf16")
    w = W.make(cfg, seed=args.seed)
    ci = W.make_conv(w, width=args.conv_width)
    Hk, Hv, dk, dv = cfg.num_qk_heads, cfg.num_v_heads, cfg.d_k, cfg.d_v
    dev = "cuda:0"
    cb = conv_bytes(cfg, w.N, w.batch, ci.width)
    R = args.layers or min(64, max(1, math.ceil(2 * MALL_BYTES / cb)))
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev).to(torch.bfloat16)
    f32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)
    offs = torch.from_numpy(w.node_offsets.astype(np.int32)).to(dev)
    par = torch.from_numpy(w.parent.astype(np.int32)).to(dev)
    sets = []
    for _ in range(R):
        sets.append(dict(
            x=bf(ci.x), ga=f32(ci.gate_a), gb=None if ci.gate_b is None else f32(ci.gate_b),
            w=f32(ci.conv_weight), b=f32(ci.conv_bias), alog=f32(ci.A_log), dtb=f32(ci.dt_bias),
            cs=bf(ci.conv_state),
            q=torch.empty((w.N, Hk, dk), device=dev, dtype=torch.bfloat16),
            k=torch.empty((w.N, Hk, dk), device=dev, dtype=torch.bfloat16),
            v=torch.empty((w.N, Hv, dv), device=dev, dtype=torch.bfloat16),
            g=torch.empty((w.N, Hv), device=dev),
            beta=torch.empty((w.N, Hv), device=dev) if cfg.mode == W.GDN else None))
    log(f"conv front end: {cfg.name} B={w.batch} N={w.N} C={2 * Hk * dk + Hv * dv} width={ci.width}, "
        f"{R} layer sets ({R * cb / 1e6:.0f} MB)")
    prob = tl.problem(w.batch, Hk, Hv, dk, dv, cfg.max_nodes, mode=cfg.mode, in_dtype=tl.BF16)
    err = torch.zeros(1, dtype=torch.int32, device=dev)

    def run(s):
        tl.conv_gates(prob, ci.width, offs, par, s["x"], s["ga"], s["gb"], s["w"], s["b"], s["alog"],
                      s["dtb"], s["cs"], s["q"], s["k"], s["v"], s["g"], s["beta"], dev_err=err)

    for _ in range(max(1, math.ceil(args.warmup / R))):
        for s in sets:
            run(s)
    torch.cuda.synchronize()
    rounds = max(1, math.ceil(args.steps / R))
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(rounds):
        for s in sets:
            run(s)
    end.record()
    torch.cuda.synchronize()
    if err.item() != 0:
        raise RuntimeError(f"device error {tl.status_string(err.item())}")
    us = start.elapsed_time(end) * 1e3 / (rounds * R)
    achieved = cb / (us * 1e-6) / 1e9
    return {
        "metric": "tree-parallel convolution front end: tree nodes/s per layer; % of HBM roofline (1 MI355X)",
        "value": round(w.N / (us * 1e-6), 1), "unit": "tree-tokens/s", "n_gpus": 1,
        "steps": rounds * R, "warmup": args.warmup, "us_per_launch": round(us, 3),
        "higher_is_better": True, "dtype": "bf16 in/out, f32 arithmetic", "data": "synthetic",
        "config": {"workload": f"{cfg.name}: B={w.batch}, {w.N} tree nodes, Hk={Hk}, Hv={Hv}, "
                               f"d_k=d_v={dk}, conv width {ci.width}", "layer_sets": R},
        "roofline": {"bound": "hbm", "kernel": "tree_conv_gates", "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "algorithmic_bytes_per_launch": int(cb)},
    }


def budget_bytes(M, B, N):
    """tree_budget_select: candidate parents and probabilities read once, rho
    and rank written once, node_offsets written, parent and src written per
    packed node (the workspace hand-off between its two launches, at most
    10 bytes per eligible candidate, stays in the caches and is not counted)."""
    return 8 * M + 8 * M + 4 * (B + 1) + 8 * N


def budget_leg(args, log):
    """Times tree_budget_select (the batch-wide allocation and the forest
    materialiser) on the candidate batch shaped after the chosen config."""
    import torch
    from paper_2608_01651_amd import treelin as tl
    from synth import workloads as W

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU (HIP) device")
    tl.lib()
    case = W.budget_case(args.workload)
    offs, par, prob = W.make_candidates(args.seed, case.sizes)
    B, M = len(case.sizes), int(offs[-1])
    dev = "cuda:0"
    i32 = dict(dtype=torch.int32, device=dev)
    t_offs = torch.from_numpy(offs.astype(np.int32)).to(dev)
    t_par = torch.from_numpy(par.astype(np.int32)).to(dev)
    t_prob = torch.from_numpy(prob.astype(np.float32)).to(dev)
    rho = torch.empty(M, dtype=torch.float32, device=dev)
    rank = torch.empty(M, **i32)
    no = torch.empty(B + 1, **i32)
    fpar = torch.empty(case.capacity, **i32)
    src = torch.empty(case.capacity, **i32)
    err = torch.zeros(1, **i32)
    prob_t = tl.problem(B, 1, 1, 16, 16, case.max_nodes)
    ws = tl.budget_workspace(B, case.max_nodes, device=dev)
    log(f"budget allocation: {args.workload} B={B} candidates={M} capacity={case.capacity} "
        f"max_nodes={case.max_nodes}")

    def run():
        tl.budget_select(prob_t, M, case.capacity, t_offs, t_par, t_prob, rho, rank, no, fpar, src, ws,
                         dev_err=err)

    for _ in range(max(1, args.warmup)):
        run()
    torch.cuda.synchronize()
    replay = run
    if args.graph:
        graph = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            run()
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph):
            run()
        torch.cuda.synchronize()
        replay = graph.replay
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        replay()
    end.record()
    torch.cuda.synchronize()
    if err.item() != 0:
        raise RuntimeError(f"device error {tl.status_string(err.item())}")
    N = int(no[-1].item())
    us = start.elapsed_time(end) * 1e3 / args.steps
    nbytes = budget_bytes(M, B, N)
    achieved = nbytes / (us * 1e-6) / 1e9
    out = {
        "metric": "batch-wide budget allocation + forest materialisation: candidates/s (1 MI355X)",
        "value": round(M / (us * 1e-6), 1), "unit": "candidates/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "us_per_allocation": round(us, 3),
        "higher_is_better": True, "dtype": "f32 scores, int32 indices", "data": "synthetic",
        "graph": bool(args.graph),
        "config": {"workload": f"{args.workload} candidate batch: B={B}, {M} candidates, "
                               f"capacity {case.capacity}, max_nodes {case.max_nodes}",
                   "selected": N},
        "roofline": {"bound": "latency", "kernel": "tree_budget_select (2 launches)",
                     "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 5), "algorithmic_bytes": int(nbytes)},
    }
    if not args.no_cpu_baseline:
        import time
        import oracle
        reps, t0 = 0, time.perf_counter()
        while time.perf_counter() - t0 < min(args.cpu_seconds, 5.0):
            oracle.budget_select(offs, par, prob, case.capacity, case.max_nodes)
            reps += 1
        dt = (time.perf_counter() - t0) / reps
        out["cpu_baseline"] = {"value": round(M / dt, 1), "unit": "candidates/s", "cores": 1,
                               "kind": "oracle", "sample": f"{reps} whole allocations of this batch"}
    return out


# ---------------------------------------------------------------------------
# CPU baseline: the fp64 oracle on a bounded sample of the same workload
# ---------------------------------------------------------------------------
_CPU_CTX = {}


def _cpu_init():
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)
    except Exception:
        pass


def _cpu_prefix(args):
    """S_pre of request b from the oracle's recurrence over its prefix."""
    cfg_name, seed, b = args
    import oracle
    from synth import workloads as W
    cfg = W.CONFIGS[cfg_name]
    if not cfg.prefix_len:
        return W.make(cfg, seed=seed, requests=[b]).state
    grp = cfg.num_v_heads // cfg.num_qk_heads
    St = None
    for c in range(W.prefix_chunks(cfg)):
        k, v, g, beta = W.prefix_chunk(cfg, seed, b, c)
        St = oracle.prefix_state(cfg.mode, k[:, np.arange(cfg.num_v_heads) // grp], v, g, beta, St0=St)
    return St[None].astype(np.float32)


def _cpu_request(args):
    cfg_name, seed, step, b, state = args
    import oracle
    from synth import workloads as W
    cfg = W.CONFIGS[cfg_name]
    w = W.make(cfg, seed=seed, step=step, requests=[b])
    oracle.verify(cfg.mode, cfg.num_qk_heads, w.node_offsets, w.parent, w.q, w.k, w.v, w.g,
                  w.beta, state, q_scale=cfg.q_scale, max_nodes=cfg.max_nodes)
    oracle.commit(cfg.mode, cfg.num_qk_heads, w.node_offsets, w.parent, w.path_offsets, w.path,
                  w.k, w.v, w.g, w.beta, state, max_nodes=cfg.max_nodes)
    return w.N


def _cpu_check(args):
    """The oracle's side of a run's check: S_pre of request b (its prefix
    recurrence), then verify and commit of b's step-0 tree from it."""
    cfg_name, seed, b = args
    import oracle
    from synth import workloads as W
    cfg = W.CONFIGS[cfg_name]
    state = _cpu_prefix((cfg_name, seed, b))
    w = W.make(cfg, seed=seed, step=0, requests=[b])
    ref_o = oracle.verify(cfg.mode, cfg.num_qk_heads, w.node_offsets, w.parent, w.q, w.k, w.v, w.g,
                          w.beta, state, q_scale=cfg.q_scale, max_nodes=cfg.max_nodes)
    ref_s = oracle.commit(cfg.mode, cfg.num_qk_heads, w.node_offsets, w.parent, w.path_offsets,
                          w.path, w.k, w.v, w.g, w.beta, state, max_nodes=cfg.max_nodes)
    return state[0].astype(np.float32), ref_o, ref_s[0]


def host_cores():
    """Host cores this job may use: the affinity mask, bounded by the job's
    share of the host where OMP_NUM_THREADS states it (one GPU's share)."""
    cores = len(os.sched_getaffinity(0))
    share = os.environ.get("OMP_NUM_THREADS", "")
    if share.isdigit() and int(share) > 0:
        cores = min(cores, int(share))
    return max(1, cores)


def cpu_leg(args, cfg, check_names, log):
    """Everything that runs the oracle, before the GPU is touched (the worker
    pool forks): the oracle's side of each workload's check, and the CPU
    baseline of the headline workload."""
    import concurrent.futures as cf
    import multiprocessing as mp
    from synth import workloads as W
    cores = host_cores()
    ctx = mp.get_context("fork")
    checks = {}
    cpu = None
    with cf.ProcessPoolExecutor(max_workers=cores, mp_context=ctx, initializer=_cpu_init) as ex:
        t0 = time.perf_counter()
        jobs = {n: (sample_requests(W.CONFIGS[n]),
                    [ex.submit(_cpu_check, (n, args.seed, b)) for b in sample_requests(W.CONFIGS[n])])
                for n in check_names}
        for n, (sample, futs) in jobs.items():
            res = [f.result() for f in futs]
            checks[n] = {"sample": sample,
                         "state_pre": np.stack([r[0] for r in res]),
                         "ref_out": np.concatenate([r[1] for r in res]),
                         "ref_state": np.stack([r[2] for r in res])}
        log(f"oracle checks of {', '.join(check_names)} prepared in {time.perf_counter() - t0:.1f} s")
        if not args.no_cpu_baseline:
            cpu = cpu_baseline(args, cfg, log, ex, cores)
    if cpu is not None:
        cpu["single_core"] = cpu_single_core(args, cfg, log)
    return checks, cpu


def cpu_baseline(args, cfg, log, ex, cores):
    """The fp64 oracle on a bounded sample: whole steps of up to 32 requests
    of the same workload (each step draws new trees; a request's S_pre is its
    prefix state), repeated until about args.cpu_seconds of wall time, one
    process per core."""
    reqs = list(range(min(cfg.batch, 32)))
    states = list(ex.map(_cpu_prefix, [(cfg.name, args.seed, b) for b in reqs]))
    # the timed region covers drawing each request's tree inputs (cheap)
    # and the oracle's verify + commit of it
    t0 = time.perf_counter()
    nodes = steps = 0
    while True:
        nodes += sum(ex.map(_cpu_request, [(cfg.name, args.seed, steps, b, states[b]) for b in reqs]))
        steps += 1
        dt = time.perf_counter() - t0
        if dt >= args.cpu_seconds or steps >= 256:
            break
    log(f"oracle: {nodes} nodes in {steps} steps of {len(reqs)} requests, {dt:.2f} s on {cores} processes")
    cpu_model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    _CPU_CTX["states"] = states
    return {"value": nodes / dt, "unit": "tree-tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"fp64 oracle verify+commit of {steps} steps x requests 0..{len(reqs) - 1} of the "
                      f"{cfg.name} workload ({nodes} tree nodes), one process per core, "
                      f"{dt:.2f} s wall; CPU: {cpu_model}; cores = the affinity mask bounded by the "
                      f"job's host share (OMP_NUM_THREADS)"}


def cpu_single_core(args, cfg, log):
    """The same oracle work on one core: whole requests of step 0 in order,
    for about a quarter of args.cpu_seconds."""
    _cpu_init()
    states = _CPU_CTX.get("states") or []
    t0 = time.perf_counter()
    nodes = reqs = 0
    while reqs < len(states):
        nodes += _cpu_request((cfg.name, args.seed, 0, reqs, states[reqs]))
        reqs += 1
        if time.perf_counter() - t0 >= args.cpu_seconds / 4:
            break
    dt = time.perf_counter() - t0
    log(f"oracle on one core: {nodes} nodes ({reqs} requests) in {dt:.2f} s")
    return {"value": nodes / dt if dt > 0 else None, "unit": "tree-tokens/s", "cores": 1,
            "sample": f"requests 0..{reqs - 1} of step 0 ({nodes} tree nodes), {dt:.2f} s"}


def copy_bandwidth():
    """A plain device-to-device copy of 512 MiB (torch copy_): bytes copied,
    ms per copy and read + write GB/s.  It is the reference kernel for scaling
    rocprofv3's FETCH_SIZE / WRITE_SIZE and the achievable copy bandwidth."""
    import torch
    n = (512 << 20) // 4
    src = torch.empty(n, dtype=torch.float32, device="cuda:0").uniform_()
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 10
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    nbytes = src.numel() * 4
    del src, dst
    return nbytes, ms, 2 * nbytes / (ms * 1e-3) / 1e9


def calibrate_copy(log):
    nbytes, ms, gbs = copy_bandwidth()
    log(f"copy of {nbytes >> 20} MiB: {ms * 1e3:.1f} us, {gbs:.0f} GB/s read+write")
    print(json.dumps({"copy_bytes": nbytes, "copy_us": round(ms * 1e3, 2),
                      "copy_gbs": round(gbs, 1)}), flush=True)


def traffic_for(cfg_name, kernel):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they
    were taken on the current kernel sources."""
    p = os.path.join(ROOT, "profiles", f"traffic_{cfg_name}.json")
    try:
        d = json.load(open(p))
    except (OSError, ValueError):
        return None
    if d.get("src_hash") != source_hash() or kernel not in d:
        return None
    return d[kernel].get("bytes_per_launch")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=40)
    ap.add_argument("--workload", default="production",
                    choices=["tiny", "mid", "production", "gdn", "large"])
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--layers", type=int, default=0, help="layer buffer sets (0: auto)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="wall time of the oracle sample (whole steps)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--conv", action="store_true",
                    help="time the tree-parallel convolution front end (tree_conv_gates) instead")
    ap.add_argument("--conv-width", type=int, default=4)
    ap.add_argument("--budget", action="store_true",
                    help="time the batch-wide budget allocation (tree_budget_select) instead")
    ap.add_argument("--graph", action="store_true",
                    help="capture one round of launches in a HIP graph and time its replays")
    ap.add_argument("--commit-layers", action="store_true",
                    help="commit every layer set with one tree_state_commit_layers call")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the gdn and large workloads that follow the headline one")
    ap.add_argument("--extra-steps", type=int, default=60,
                    help="timed steps of each extra workload")
    ap.add_argument("--no-check", action="store_true",
                    help="skip the oracle check of a sampled step")
    ap.add_argument("--quiet", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only time a plain 512 MiB device copy (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(every (request, head) unit is independent, so the path shards over requests "
              "or head groups without communication).", file=sys.stderr)
        sys.exit(2)

    def log(msg):
        if not args.quiet:
            print(f"[bench] {msg}", file=sys.stderr, flush=True)

    if args.calibrate_copy:
        calibrate_copy(log)
        return
    from synth import workloads as W
    cfg = W.CONFIGS[args.workload]
    if args.conv:
        print(json.dumps(conv_leg(args, cfg, log)), flush=True)
        return
    if args.budget:
        print(json.dumps(budget_leg(args, log)), flush=True)
        return
    extra = [] if args.no_extra else [n for n in ("gdn", "large") if n != cfg.name]
    check_names = [] if args.no_check else [cfg.name] + extra
    # the oracle's work first, before the GPU is touched, so the pool may fork
    checks, cpu = cpu_leg(args, cfg, check_names, log)
    g = gpu_leg(args, cfg, log, check=checks.get(cfg.name))
    line = summarize(cfg, g, args)
    _, _, copy_gbs = copy_bandwidth()   # context only: the roofline is the 8 TB/s peak
    path_gbs = line["path_hbm_frac"] * HBM_PEAK_GBS
    line["copy_context"] = {"copy_gbs": round(copy_gbs, 1), "path_frac_of_copy": round(path_gbs / copy_gbs, 4),
                            "note": "a 512 MiB device copy in the same run (read + write bytes / time)"}
    line["cpu_baseline"] = cpu
    line["paper_context"] = PAPER_CONTEXT
    if extra:
        line["workloads"] = {}
        for n in extra:
            c = W.CONFIGS[n]
            ge = gpu_leg(args, c, log, check=checks.get(n), steps=args.extra_steps,
                         warmup=min(args.warmup, args.extra_steps))
            sub = summarize(c, ge, args)
            line["workloads"][n] = {k: sub[k] for k in (
                "value", "unit", "ms_per_step", "steps", "verify_us", "commit_us", "path_hbm_frac",
                "roofline", "check", "config")}
    print(json.dumps(line), flush=True)


PAPER_CONTEXT = {
    "what": "the paper's per-layer GDN tree-verification latency (Table kernel-verify, §6.5): Qwen3.5-9B "
            "GDN layers, drafter top-k 4 and depth 8, tree size not stated, kernel precision not stated; "
            "other hardware, context only (not this workload, not the target)",
    "rows": [
        {"hardware": "A100 80GB SXM4 (2.04 TB/s HBM2e)", "batch": 1, "serial_us": 174, "paper_us": 50.6},
        {"hardware": "A100 80GB SXM4 (2.04 TB/s HBM2e)", "batch": 16, "serial_us": 822, "paper_us": 110},
        {"hardware": "GB10 / DGX Spark (273 GB/s LPDDR5x)", "batch": 1, "serial_us": 333, "paper_us": 66.6},
        {"hardware": "GB10 / DGX Spark (273 GB/s LPDDR5x)", "batch": 16, "serial_us": 3420, "paper_us": 443},
    ],
}

DTYPE = ("f32: fp32 state, gates, accumulation and output; bf16 q/k/v; contractions on bf16 MFMA "
         "with each fp32 operand split into bf16 hi + lo (about 2^-16 relative)")


def summarize(cfg, g, args):
    """The bench line's fields for one workload's GPU leg."""
    w = g["w"]
    ms_step = g["total_ms"] / g["steps"]
    value = w.N / (ms_step * 1e-3)
    path_gbs = (g["verify_bytes"] + g["commit_bytes"]) / (ms_step * 1e-3) / 1e9
    kern = {"verify": (g["verify_ms"], g["verify_bytes"]), "commit": (g["commit_ms"], g["commit_bytes"])}
    dom = max(kern, key=lambda k: kern[k][0])
    dom_ms, dom_bytes = kern[dom]
    achieved = dom_bytes / (dom_ms * 1e-3) / 1e9
    roofline = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": traffic_for(cfg.name, dom),
                "algorithmic_bytes_per_launch": int(dom_bytes),
                "launch_us": round(dom_ms * 1e3, 3),
                "timing": f"{dom}'s launches back to back over the layer sets, one event before and "
                          f"one after, divided by the launch count"}
    return {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "tree-tokens/s",
        "n_gpus": 1,
        "steps": g["steps"],
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": DTYPE,
        "data": "synthetic",
        "config": {
            "workload": f"{cfg.name}: B={w.batch}, Hk={cfg.num_qk_heads}, Hv={cfg.num_v_heads}, "
                        f"d_k=d_v={cfg.d_k}, {'gated delta rule' if cfg.mode else 'gated linear attention'}, "
                        f"{w.N} tree nodes, {cfg.in_dtype} q/k/v, fp32 state and output",
            "batch": w.batch, "tree_nodes": w.N, "accepted_rows": int(w.path.size),
            "in_dtype": cfg.in_dtype, "layer_sets": g["R"], "parallelism": "none (1 GPU)",
        },
        "timing": ("value and ms_per_step from replays of a captured HIP graph of one round; "
                   if args.graph else
                   "value and ms_per_step from one pass with an event before and after the timed steps; ")
                  + "verify_us and commit_us from each kernel's launches alone, back to back, "
                    "an event before and after",
        "verify_us": round(g["verify_ms"] * 1e3, 3),
        "commit_us": round(g["commit_ms"] * 1e3, 3),
        "commit_call": "tree_state_commit_layers (all layer sets)" if args.commit_layers
                       else "tree_state_commit (one per layer set)",
        "path_hbm_frac": round(path_gbs / HBM_PEAK_GBS, 4),
        "roofline": roofline,
        "check": g["check"],
    }


if __name__ == "__main__":
    main()
