"""HIP-graph capture of a verification round in a capacity bucket (§5.2:
captured graphs keep fixed addresses and kernel shapes while the tree
topology varies from round to round).

A bucket fixes the batch size, max_nodes and the buffers.  Every kernel
reads the request sizes, parents and paths from device memory, so one
captured graph of verify -> commit (and of the unified commit) replays
correctly for any forest that fits the bucket: fewer nodes per request,
different shapes, requests with no nodes.  Each round below writes a new
forest into the same buffers with ordinary eager copies, replays the graph,
and checks the replay against eager launches of the same calls and against
the fp64 oracle.  The graph holds kernels only (no memset nodes)."""
import numpy as np
import pytest
import torch

import oracle
from synth import workloads as W
from tests import gpu_helpers as H
from paper_2608_01651_amd import treelin as tl

pytestmark = pytest.mark.gpu


def bucket_round(cfg, B, cap, rnd):
    """A forest of up to B requests (some empty) and at most cap nodes in all."""
    rng = np.random.default_rng([rnd, 77])
    w = W.make(cfg, step=rnd, requests=list(range(B)))
    sizes = np.diff(w.node_offsets).copy()
    keep = []
    for b in range(B):
        T = int(sizes[b])
        if rnd % 2 == 1 and b % 3 == 2:
            keep.append(0)                               # an empty request
        else:
            keep.append(int(rng.integers(max(1, T // 2), T + 1)))
    # truncate every tree to its first keep[b] nodes (still parent-before-child)
    parts = {k: [] for k in ("parent", "q", "k", "v", "g", "beta", "path")}
    offs, poffs = [0], [0]
    for b in range(B):
        o, T = int(w.node_offsets[b]), keep[b]
        parts["parent"].append(w.parent[o:o + T])
        for key in ("q", "k", "v", "g"):
            parts[key].append(getattr(w, key)[o:o + T])
        if w.beta is not None:
            parts["beta"].append(w.beta[o:o + T])
        p = w.path[w.path_offsets[b]:w.path_offsets[b + 1]]
        p = p[p < T] if T else p[:0]
        # the path must stay a root-first chain: keep its prefix of kept nodes
        good = 0
        while good < len(p) and p[good] < T:
            good += 1
        parts["path"].append(p[:good])
        offs.append(offs[-1] + T)
        poffs.append(poffs[-1] + good)
    N = offs[-1]
    assert N <= cap
    cat = lambda key: np.concatenate(parts[key]) if parts[key] else None
    return dict(node_offsets=np.asarray(offs, np.int32), parent=cat("parent").astype(np.int32),
                q=cat("q"), k=cat("k"), v=cat("v"), g=cat("g"),
                beta=cat("beta") if w.beta is not None else None,
                path_offsets=np.asarray(poffs, np.int32), path=cat("path").astype(np.int32), N=N)


@pytest.mark.parametrize("name", ["mid", "production", "gdn"])
def test_graph_replay_across_topologies(name):
    cfg = W.CONFIGS[name]
    B = 3
    cap = B * cfg.max_nodes
    Hk, Hv, dk, dv = cfg.num_qk_heads, cfg.num_v_heads, cfg.d_k, cfg.d_v
    dev = H.dev()
    dt = torch.float32 if cfg.in_dtype == "f32" else torch.bfloat16
    buf = dict(node_offsets=torch.zeros(B + 1, dtype=torch.int32, device=dev),
               parent=torch.zeros(cap, dtype=torch.int32, device=dev),
               q=torch.zeros((cap, Hk, dk), dtype=dt, device=dev),
               k=torch.zeros((cap, Hk, dk), dtype=dt, device=dev),
               v=torch.zeros((cap, Hv, dv), dtype=dt, device=dev),
               g=torch.zeros((cap, Hv), device=dev),
               beta=torch.zeros((cap, Hv), device=dev) if cfg.mode == W.GDN else None,
               path_offsets=torch.zeros(B + 1, dtype=torch.int32, device=dev),
               path=torch.zeros(cap, dtype=torch.int32, device=dev),
               state=torch.zeros((B, Hv, dv, dk), device=dev),
               out=torch.zeros((cap, Hv, dv), device=dev),
               err=torch.zeros(1, dtype=torch.int32, device=dev))
    prob = H.problem_for(cfg, B)

    def enqueue(b):
        tl.verify(prob, b["node_offsets"], b["parent"], b["q"], b["k"], b["v"], b["g"], b["beta"],
                  b["state"], b["out"], dev_err=b["err"])
        tl.commit(prob, b["node_offsets"], b["parent"], b["path_offsets"], b["path"], b["k"], b["v"],
                  b["g"], b["beta"], b["state"], dev_err=b["err"])

    def load(b, r, state0):
        b["node_offsets"].copy_(torch.from_numpy(r["node_offsets"]))
        b["path_offsets"].copy_(torch.from_numpy(r["path_offsets"]))
        n = r["N"]
        if n:
            b["parent"][:n].copy_(torch.from_numpy(r["parent"]))
            for key in ("q", "k", "v", "g"):
                b[key][:n].copy_(torch.from_numpy(np.ascontiguousarray(r[key])).to(b[key].dtype))
            if b["beta"] is not None:
                b["beta"][:n].copy_(torch.from_numpy(r["beta"]))
        if r["path"].size:
            b["path"][:r["path"].size].copy_(torch.from_numpy(r["path"]))
        b["state"].copy_(state0)
        b["out"].fill_(float("nan"))
        b["err"].zero_()

    state0 = torch.from_numpy((0.3 * np.random.default_rng(1).standard_normal((B, Hv, dv, dk)))
                              .astype(np.float32)).to(dev)
    # capture once, on a side stream, after a warm-up on it
    r0 = bucket_round(cfg, B, cap, 0)
    load(buf, r0, state0)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        enqueue(buf)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        enqueue(buf)
    torch.cuda.synchronize()

    eager = {key: (t.clone() if t is not None else None) for key, t in buf.items()}
    for rnd in range(1, 5):
        r = bucket_round(cfg, B, cap, rnd)
        load(buf, r, state0)
        graph.replay()
        torch.cuda.synchronize()
        load(eager, r, state0)                            # the same round, launched eagerly
        enqueue(eager)
        torch.cuda.synchronize()
        assert buf["err"].item() == 0 and eager["err"].item() == 0
        n = r["N"]
        assert torch.equal(buf["out"][:n], eager["out"][:n]), f"round {rnd}: replay differs from eager"
        assert torch.equal(buf["state"], eager["state"]), f"round {rnd}: committed state differs"
        if rnd > 1:
            continue                                      # the oracle once (it is slow)
        ref_o = oracle.verify(cfg.mode, Hk, r["node_offsets"], r["parent"], r["q"], r["k"], r["v"],
                              r["g"], r["beta"], state0.cpu().numpy(), q_scale=cfg.q_scale,
                              max_nodes=cfg.max_nodes)
        assert H.slice_rel_err(buf["out"][:n].cpu().numpy(), ref_o, r["node_offsets"]) < H.TOL
        ref_s = oracle.commit(cfg.mode, Hk, r["node_offsets"], r["parent"], r["path_offsets"], r["path"],
                              r["k"], r["v"], r["g"], r["beta"], state0.cpu().numpy(),
                              max_nodes=cfg.max_nodes)
        assert H.state_rel_err(buf["state"].cpu().numpy(), ref_s) < H.TOL


def test_graph_replay_unified_commit():
    """The unified commit of two layers, captured once and replayed over
    rounds with new trees and terminals."""
    cfg = W.CONFIGS["gdn"]
    B, L = 3, 2
    cap = B * cfg.max_nodes
    Hk, Hv, dk, dv = cfg.num_qk_heads, cfg.num_v_heads, cfg.d_k, cfg.d_v
    dev = H.dev()
    rng = np.random.default_rng(3)
    offs = torch.zeros(B + 1, dtype=torch.int32, device=dev)
    par = torch.zeros(cap, dtype=torch.int32, device=dev)
    term = torch.zeros(B, dtype=torch.int32, device=dev)
    lay = [dict(k=torch.zeros((cap, Hk, dk), dtype=torch.bfloat16, device=dev),
                v=torch.zeros((cap, Hv, dv), dtype=torch.bfloat16, device=dev),
                g=torch.zeros((cap, Hv), device=dev), beta=torch.zeros((cap, Hv), device=dev),
                state=torch.zeros((B, Hv, dv, dk), device=dev)) for _ in range(L)]
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    prob = H.problem_for(cfg, B)
    table = [tl.layer(x["k"], x["v"], x["g"], x["beta"], x["state"]) for x in lay]
    states0 = [(0.3 * rng.standard_normal((B, Hv, dv, dk))).astype(np.float32) for _ in range(L)]

    def enqueue():
        tl.commit_layers(prob, table, offs, par, term, dev_err=err)

    def load(rnd):
        w = W.make(cfg, step=rnd, requests=[0, 1, 2])
        offs.copy_(torch.from_numpy(w.node_offsets))
        par[:w.N].copy_(torch.from_numpy(w.parent))
        t = []
        for b in range(B):
            p0, p1 = int(w.path_offsets[b]), int(w.path_offsets[b + 1])
            t.append(int(w.path[p1 - 1]) if p1 > p0 and not (rnd == 2 and b == 1) else -1)
        term.copy_(torch.tensor(t, dtype=torch.int32))
        for l, x in enumerate(lay):
            lrng = np.random.default_rng([rnd, l])
            vals = dict(k=W.round_bf16(w.k + 0.1 * l), v=W.round_bf16(w.v * (1 + l)),
                        g=w.g - 0.05 * l, beta=w.beta)
            for key in ("k", "v"):
                x[key][:w.N].copy_(torch.from_numpy(np.ascontiguousarray(vals[key])).to(torch.bfloat16))
            for key in ("g", "beta"):
                x[key][:w.N].copy_(torch.from_numpy(np.ascontiguousarray(vals[key], dtype=np.float32)))
            x["state"].copy_(torch.from_numpy(states0[l]))
            x["vals"] = vals
        err.zero_()
        return w, t

    load(0)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        enqueue()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        enqueue()
    torch.cuda.synchronize()
    for rnd in range(1, 4):
        w, t = load(rnd)
        graph.replay()
        torch.cuda.synchronize()
        assert err.item() == 0
        ref = oracle.commit_layers(cfg.mode, Hk, w.node_offsets, w.parent, t,
                                   [(x["vals"]["k"], x["vals"]["v"], x["vals"]["g"], x["vals"]["beta"], s0)
                                    for x, s0 in zip(lay, states0)], max_nodes=cfg.max_nodes)
        for l, x in enumerate(lay):
            assert H.state_rel_err(x["state"].cpu().numpy(), ref[l]) < H.TOL, (rnd, l)
