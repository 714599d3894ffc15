"""GPU edge cases through the C ABI, against the fp64 oracle: device error
reporting (the bad request is skipped, the others are computed), empty
paths and requests, slot indirection, determinism, several verify -> commit
steps with carried state, other head dimensions and group sizes, forests
with several roots, the deepest tree (a 256-node chain), a query scale, and
the full production batch in the benchmark's launch configuration."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from synth import workloads as W
from tests import gpu_helpers as H
from paper_2608_01651_amd import treelin as tl

pytestmark = pytest.mark.gpu


def cfg_of(base, **kw):
    return dataclasses.replace(W.CONFIGS[base], **kw)


def custom(cfg, parents, paths, seed=0):
    """A workload over explicit forests: q/k unit rows, v ~ N(0,1), gates and
    beta drawn like the configuration's, stored in its input dtype."""
    rng = np.random.default_rng([seed, 4242])
    Hk, Hv, dk, dv = cfg.num_qk_heads, cfg.num_v_heads, cfg.d_k, cfg.d_v
    sizes = [len(p) for p in parents]
    N = int(sum(sizes))

    def store(x):
        x = np.asarray(x, np.float32)
        return W.round_bf16(x) if cfg.in_dtype == "bf16" else x

    def unit(shape):
        x = rng.standard_normal(shape)
        return store(x / np.linalg.norm(x, axis=-1, keepdims=True))

    g = (-np.logaddexp(0.0, rng.standard_normal((N, Hv)) - cfg.gate_shift)).astype(np.float32)
    beta = None
    if cfg.mode == W.GDN:
        beta = (1.0 / (1.0 + np.exp(-rng.standard_normal((N, Hv))))).astype(np.float32)
    return W.Workload(
        cfg=cfg, seed=seed, step=0,
        node_offsets=np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32),
        parent=np.concatenate([np.asarray(p, np.int32) for p in parents]) if N else np.zeros(0, np.int32),
        q=unit((N, Hk, dk)), k=unit((N, Hk, dk)), v=store(rng.standard_normal((N, Hv, dv))),
        g=g, beta=beta,
        path_offsets=np.concatenate([[0], np.cumsum([len(p) for p in paths])]).astype(np.int32),
        path=np.concatenate([np.asarray(p, np.int32) for p in paths]) if sum(map(len, paths))
        else np.zeros(0, np.int32),
        state=None)


def rand_state(cfg, slots, seed=0, scale=0.3):
    rng = np.random.default_rng([seed, 777])
    return (scale * rng.standard_normal((slots, cfg.num_v_heads, cfg.d_v, cfg.d_k))).astype(np.float32)


def o_verify(cfg, w, state, slot=None, max_nodes=None):
    return oracle.verify(cfg.mode, cfg.num_qk_heads, w.node_offsets, w.parent, w.q, w.k, w.v, w.g,
                         w.beta, state, slot=slot, q_scale=cfg.q_scale,
                         max_nodes=max_nodes or cfg.max_nodes)


def o_commit(cfg, w, state, slot=None, max_nodes=None):
    return oracle.commit(cfg.mode, cfg.num_qk_heads, w.node_offsets, w.parent, w.path_offsets,
                         w.path, w.k, w.v, w.g, w.beta, state, slot=slot,
                         max_nodes=max_nodes or cfg.max_nodes)


def sub(w, keep):
    """Requests `keep` of w as a workload of their own (for oracle references)."""
    reqs = []
    for b in keep:
        o0, o1 = int(w.node_offsets[b]), int(w.node_offsets[b + 1])
        p0, p1 = int(w.path_offsets[b]), int(w.path_offsets[b + 1])
        reqs.append((o0, o1, p0, p1))
    cat = lambda x: np.concatenate([x[o0:o1] for o0, o1, _, _ in reqs]) if x is not None else None
    return dataclasses.replace(
        w, node_offsets=np.concatenate([[0], np.cumsum([o1 - o0 for o0, o1, _, _ in reqs])]).astype(np.int32),
        parent=cat(w.parent), q=cat(w.q), k=cat(w.k), v=cat(w.v), g=cat(w.g), beta=cat(w.beta),
        path_offsets=np.concatenate([[0], np.cumsum([p1 - p0 for _, _, p0, p1 in reqs])]).astype(np.int32),
        path=np.concatenate([w.path[p0:p1] for _, _, p0, p1 in reqs]).astype(np.int32))


def rows_of(w, keep):
    return np.concatenate([np.arange(w.node_offsets[b], w.node_offsets[b + 1]) for b in keep])


def topk(T, seed):
    return W.topk_tree(np.random.default_rng([seed, 11]), T, (8, 4, 2), 10)


def chain_path(parent, node):
    return W.path_to(parent, node)


# ----------------------------------------------------------------------------
# device-side errors: reported once, the request skipped, the others computed
# ----------------------------------------------------------------------------

ERROR_CONFIGS = [
    ("production", dict()),                                    # <= 64 nodes, two heads per block
    ("mid", dict()),                                           # <= 64 nodes, one head per block
    ("gdn", dict(max_nodes=128)),                              # delta rule
    ("large", dict()),                                         # 65..256 nodes
    ("tiny", dict()),                                          # vector path
]


def _error_case(name, kw, T=40):
    cfg = cfg_of(name, batch=3, prefix_len=0, **kw)
    if name == "tiny":
        T = 15
    parents = [topk(T, s) if T > 15 else W.binary_tree(3) for s in range(3)]
    paths = [chain_path(p, int(np.flatnonzero(W.node_depths(p) == W.node_depths(p).max())[0]))
             for p in parents]
    return cfg, parents, paths


@pytest.mark.parametrize("name, kw", ERROR_CONFIGS)
def test_bad_parent_is_reported_and_skipped(name, kw):
    cfg, parents, paths = _error_case(name, kw)
    bad = [p.copy() for p in parents]
    bad[1][5] = 9                       # a parent after its child
    w = custom(cfg, bad, paths)
    state = rand_state(cfg, 3)
    up = H.Uploaded(w)
    got, err = H.run_verify(cfg, up, H.t_f32(state))
    assert err == tl.TL_EBADTREE
    good = [0, 2]
    ref = o_verify(cfg, sub(w, good), state[good])
    rows = rows_of(w, good)
    assert H.slice_rel_err(got[rows], ref, sub(w, good).node_offsets) <= H.TOL
    assert np.isnan(got[rows_of(w, [1])]).all(), "the bad request's rows must stay unwritten"
    st = H.t_f32(state)
    err = H.run_commit(cfg, up, st)
    assert err == tl.TL_EBADTREE
    after = st.cpu().numpy()
    np.testing.assert_array_equal(after[1], state[1])
    ref_s = o_commit(cfg, sub(w, good), state[good])
    assert H.state_rel_err(after[good], ref_s) <= H.TOL


@pytest.mark.parametrize("how", ["not_a_root", "broken_link", "out_of_range", "too_long"])
def test_bad_path_is_reported_and_slot_untouched(how):
    cfg, parents, paths = _error_case("production", {})
    paths = [list(p) for p in paths]
    if how == "not_a_root":
        paths[1] = paths[1][1:]
    elif how == "broken_link":
        paths[1] = [paths[1][0]] + paths[1][2:]
    elif how == "out_of_range":
        paths[1] = paths[1][:-1] + [len(parents[1]) + 3]
    else:
        paths[1] = list(range(len(parents[1]))) + [0]
    w = custom(cfg, parents, paths)
    state = rand_state(cfg, 3)
    st = H.t_f32(state)
    err = H.run_commit(cfg, H.Uploaded(w), st)
    assert err == tl.TL_EBADPATH
    after = st.cpu().numpy()
    np.testing.assert_array_equal(after[1], state[1])
    good = [0, 2]
    assert H.state_rel_err(after[good], o_commit(cfg, sub(w, good), state[good])) <= H.TOL


def test_tree_larger_than_max_nodes_is_reported():
    cfg = cfg_of("production", batch=2, prefix_len=0)
    w = custom(cfg, [topk(64, 1), topk(64, 2)], [[0], [0]])
    state = rand_state(cfg, 2)
    got, err = H.run_verify(cfg, H.Uploaded(w), H.t_f32(state), max_nodes=48)
    assert err == tl.TL_EBADTREE
    assert np.isnan(got).all()


# every verify kernel reads the slot map: (config, node cap, tree size)
SLOT_KERNELS = [("production", 64, 64),     # small-tree kernel
                ("gdn", 128, 100),          # dense delta-rule kernel
                ("large", 256, 200),        # large-tree kernel
                ("gdn", 144, 140),          # the delta rule tile by tile
                ("gdn", 256, 180)]          # the delta rule's per-wave path


@pytest.mark.parametrize("name, cap, T", SLOT_KERNELS)
def test_slot_out_of_range_is_reported(name, cap, T):
    cfg, parents, paths = _error_case(name, dict(max_nodes=cap), T=T)
    w = custom(cfg, parents, paths)
    state = rand_state(cfg, 4)
    slot = H.t_int([2, 4, 0])            # 4 is past the last of the 4 slots
    got, err = H.run_verify(cfg, H.Uploaded(w), H.t_f32(state), slot=slot, num_slots=4)
    assert err == tl.TL_EINVAL
    assert np.isnan(got[rows_of(w, [1])]).all()
    good = [0, 2]
    ref = o_verify(cfg, sub(w, good), state, slot=np.array([2, 0]))
    assert H.slice_rel_err(got[rows_of(w, good)], ref, sub(w, good).node_offsets) <= H.TOL


# ----------------------------------------------------------------------------
# empty paths and requests, slot indirection, determinism
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("name", ["production", "gdn", "large"])
def test_empty_paths_and_empty_requests(name):
    cfg = cfg_of(name, batch=4, prefix_len=0)
    T = {"production": 64, "gdn": 100, "large": 200}[name]
    parents = [topk(T, 1), np.zeros(0, np.int32), topk(T, 2), topk(T, 3)]
    paths = [chain_path(parents[0], T - 1), [], [], chain_path(parents[3], 7)]
    w = custom(cfg, parents, paths)
    state = rand_state(cfg, 4)
    up = H.Uploaded(w)
    got, err = H.run_verify(cfg, up, H.t_f32(state))
    assert err == 0
    assert H.slice_rel_err(got, o_verify(cfg, w, state), w.node_offsets) <= H.TOL
    st = H.t_f32(state)
    assert H.run_commit(cfg, up, st) == 0
    after = st.cpu().numpy()
    np.testing.assert_array_equal(after[1], state[1])     # no nodes, no path
    np.testing.assert_array_equal(after[2], state[2])     # empty path
    assert H.state_rel_err(after, o_commit(cfg, w, state)) <= H.TOL


@pytest.mark.parametrize("name, cap, T", SLOT_KERNELS)
def test_slot_indirection(name, cap, T):
    cfg = cfg_of(name, batch=3, prefix_len=0, max_nodes=cap)
    parents = [topk(T, s) for s in range(3)]
    paths = [chain_path(p, 20) for p in parents]
    w = custom(cfg, parents, paths)
    state = rand_state(cfg, 5)
    slot_np = np.array([4, 0, 2], np.int32)
    up = H.Uploaded(w)
    got, err = H.run_verify(cfg, up, H.t_f32(state), slot=H.t_int(slot_np), num_slots=5)
    assert err == 0
    assert H.slice_rel_err(got, o_verify(cfg, w, state, slot=slot_np), w.node_offsets) <= H.TOL
    st = H.t_f32(state)
    assert H.run_commit(cfg, up, st, slot=H.t_int(slot_np), num_slots=5) == 0
    after = st.cpu().numpy()
    ref = o_commit(cfg, w, state, slot=slot_np)
    assert H.state_rel_err(after, ref) <= H.TOL
    np.testing.assert_array_equal(after[[1, 3]], state[[1, 3]])   # slots no request names


@pytest.mark.parametrize("name", ["production", "gdn", "large"])
def test_deterministic(name):
    cfg = cfg_of(name, prefix_len=0)
    w = W.make(cfg, requests=[0, 1, 2])
    state = rand_state(cfg, 3)
    up = H.Uploaded(w)
    a, _ = H.run_verify(cfg, up, H.t_f32(state))
    b, _ = H.run_verify(cfg, up, H.t_f32(state))
    np.testing.assert_array_equal(a, b)
    s1, s2 = H.t_f32(state), H.t_f32(state)
    H.run_commit(cfg, up, s1)
    H.run_commit(cfg, up, s2)
    np.testing.assert_array_equal(s1.cpu().numpy(), s2.cpu().numpy())


# ----------------------------------------------------------------------------
# several steps: verify, commit, next step's trees on the committed state
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("name, reqs", [("large", [0, 1, 5]), ("gdn", [0, 1]), ("production", [0, 7])])
def test_three_steps_with_carried_state(name, reqs):
    cfg = cfg_of(name, prefix_len=0)
    state = rand_state(cfg, len(reqs), scale=0.1)
    st = H.t_f32(state)
    ref_state = state.astype(np.float64)
    for step in range(3):
        w = W.make(cfg, step=step, requests=reqs)
        up = H.Uploaded(w)
        got, err = H.run_verify(cfg, up, st)
        assert err == 0
        ref = o_verify(cfg, w, ref_state)
        e = H.slice_rel_err(got, ref, w.node_offsets)
        assert e <= H.TOL, (step, e)
        assert H.run_commit(cfg, up, st) == 0
        ref_state = o_commit(cfg, w, ref_state)
        e = H.state_rel_err(st.cpu().numpy(), ref_state)
        assert e <= H.TOL, (step, e)


# ----------------------------------------------------------------------------
# shapes: head dimensions, group sizes, forests, the deepest tree, q scale
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("d", [16, 32, 64, 128])
@pytest.mark.parametrize("hk, hv", [(2, 4), (3, 3), (1, 4)])
@pytest.mark.parametrize("mode", [W.GLA, W.GDN])
def test_head_dims_and_groups(d, hk, hv, mode):
    cfg = cfg_of("production" if mode == W.GLA else "gdn", batch=3, num_qk_heads=hk, num_v_heads=hv,
                 d_k=d, d_v=d, prefix_len=0, max_nodes=64)
    parents = [topk(64, 1), topk(37, 2), topk(16, 3)]
    paths = [chain_path(p, len(p) - 1) for p in parents]
    w = custom(cfg, parents, paths)
    state = rand_state(cfg, 3)
    up = H.Uploaded(w)
    got, err = H.run_verify(cfg, up, H.t_f32(state))
    assert err == 0
    e = H.slice_rel_err(got, o_verify(cfg, w, state), w.node_offsets)
    assert e <= H.TOL, e
    st = H.t_f32(state)
    assert H.run_commit(cfg, up, st) == 0
    assert H.state_rel_err(st.cpu().numpy(), o_commit(cfg, w, state)) <= H.TOL


@pytest.mark.parametrize("seed", range(12))
def test_commit_random_batches(seed):
    """Commit over random batches whose slot counts fall in each split of the
    launch (under 512 slots: four workgroups per slot; under 1024: two; more:
    one), for both rules, several head dimensions and group sizes, with empty
    and long accepted paths."""
    rng = np.random.default_rng([seed, 91])
    mode = W.GDN if seed % 2 else W.GLA
    d = int(rng.choice([32, 64, 128]))
    hk = int(rng.choice([1, 2, 4]))
    hv = hk * int(rng.choice([1, 2]))
    B = int(rng.choice([3, 60, 150, 320]))
    cfg = cfg_of("gdn" if mode == W.GDN else "production", batch=B, num_qk_heads=hk, num_v_heads=hv,
                 d_k=d, d_v=d, prefix_len=0, max_nodes=64)
    parents, paths = [], []
    for b in range(B):
        T = int(rng.integers(1, 65))
        p = _multi_root(T, int(rng.integers(1, 3)), 1000 * seed + b)
        parents.append(p)
        node = int(rng.integers(-1, T))   # -1: nothing accepted
        paths.append([] if node < 0 else chain_path(p, node))
    w = custom(cfg, parents, paths, seed=seed)
    state = rand_state(cfg, B, seed=seed)
    up = H.Uploaded(w)
    print(f"commit random seed={seed} mode={mode} d={d} Hk={hk} Hv={hv} B={B} slots={B * hv}", flush=True)
    st = H.t_f32(state)
    assert H.run_commit(cfg, up, st) == 0
    assert H.state_rel_err(st.cpu().numpy(), o_commit(cfg, w, state)) <= H.TOL


@pytest.mark.parametrize("seed", range(8))
def test_verify_random_batches(seed):
    """Verify over random batches that reach every kernel of the dispatch:
    buckets of 64, 128 and 256 nodes (the small-tree kernel, the tile walk with
    2 and 4 mask words, and the delta rule's kernel for node caps above 160 at d = 128),
    both rules, d = 32, 64 and 128, ragged trees with one to three roots."""
    rng = np.random.default_rng([seed, 93])
    mode = W.GDN if seed % 2 else W.GLA
    d = int(rng.choice([32, 64, 128]))
    max_nodes = int(rng.choice([64, 128, 256]))
    if seed == 7:   # one delta-rule draw on the kernel for node caps above 160 at d = 128
        d, max_nodes = 128, 256
    B = int(rng.integers(1, 5))
    cfg = cfg_of("gdn" if mode == W.GDN else "production", batch=B, num_qk_heads=2, num_v_heads=4,
                 d_k=d, d_v=d, prefix_len=0, max_nodes=max_nodes)
    parents = [_multi_root(int(rng.integers(1, max_nodes + 1)), int(rng.integers(1, 4)), 2000 * seed + b)
               for b in range(B)]
    paths = [chain_path(p, len(p) - 1) for p in parents]
    w = custom(cfg, parents, paths, seed=seed)
    state = rand_state(cfg, B, seed=seed)
    up = H.Uploaded(w)
    print(f"verify random seed={seed} mode={mode} d={d} max_nodes={max_nodes} sizes={[len(p) for p in parents]}",
          flush=True)
    got, err = H.run_verify(cfg, up, H.t_f32(state))
    assert err == 0
    assert H.slice_rel_err(got, o_verify(cfg, w, state), w.node_offsets) <= H.TOL


def _multi_root(T, roots, seed):
    rng = np.random.default_rng([seed, 5])
    p = np.empty(T, np.int32)
    p[:roots] = -1
    for i in range(roots, T):
        p[i] = rng.integers(0, i)
    return p


@pytest.mark.parametrize("name, T", [("production", 40), ("production", 64), ("gdn", 128),
                                     ("large", 256), ("tiny", 12)])
def test_forests_with_several_roots(name, T):
    cfg = cfg_of(name, batch=2, prefix_len=0, max_nodes=max(T, W.CONFIGS[name].max_nodes))
    parents = [_multi_root(T, 3, 1), _multi_root(T, 5, 2)]
    paths = [chain_path(parents[0], T - 1), chain_path(parents[1], T // 2)]
    w = custom(cfg, parents, paths)
    state = rand_state(cfg, 2)
    up = H.Uploaded(w)
    got, err = H.run_verify(cfg, up, H.t_f32(state))
    assert err == 0
    assert H.slice_rel_err(got, o_verify(cfg, w, state), w.node_offsets) <= H.TOL
    st = H.t_f32(state)
    assert H.run_commit(cfg, up, st) == 0
    assert H.state_rel_err(st.cpu().numpy(), o_commit(cfg, w, state)) <= H.TOL


@pytest.mark.parametrize("d, max_nodes, sizes", [(128, 144, [144, 129, 40]), (128, 160, [160, 131, 90]),
                                                  (64, 256, [256, 230, 100])])
def test_tile_walk_delta_rule_single_buffer(d, max_nodes, sizes):
    """The delta rule where the tile walk's layout fits LDS only with one chunk
    buffer (node caps of 144 and 160 at d = 128, 256 at d = 64): the value work
    and the chunks of the next tile alternate between barriers.  Ragged
    multi-root trees, verify and commit."""
    cfg = cfg_of("gdn", batch=len(sizes), num_qk_heads=2, num_v_heads=4, d_k=d, d_v=d,
                 prefix_len=0, max_nodes=max_nodes)
    parents = [_multi_root(T, 1 + k, 30 + k) for k, T in enumerate(sizes)]
    paths = [chain_path(p, len(p) - 1) for p in parents]
    w = custom(cfg, parents, paths, seed=d + max_nodes)
    state = rand_state(cfg, len(sizes), seed=7)
    up = H.Uploaded(w)
    print(f"single-buffer tile walk d={d} max_nodes={max_nodes} sizes={sizes}", flush=True)
    got, err = H.run_verify(cfg, up, H.t_f32(state))
    assert err == 0
    assert H.slice_rel_err(got, o_verify(cfg, w, state), w.node_offsets) <= H.TOL
    st = H.t_f32(state)
    assert H.run_commit(cfg, up, st) == 0
    assert H.state_rel_err(st.cpu().numpy(), o_commit(cfg, w, state)) <= H.TOL


def test_delta_rule_dense_kernel_tile_counts():
    """The delta rule's dense kernel (d = 128, node cap 128) has branch-free
    code for trees that fill all 8 node tiles (113..128 nodes) and, when
    every row of the last tile is a node (128 nodes), for the readout too;
    other trees take the generic code.  One batch with trees of 128, 127,
    120 and 113 nodes (full tiles, the last one ragged), 112 and 40 (fewer
    tiles), branching and multi-root, verify and commit."""
    cfg = cfg_of("gdn", batch=6, num_qk_heads=2, num_v_heads=4, d_k=128, d_v=128,
                 prefix_len=0, max_nodes=128)
    parents = [_multi_root(128, 1, 70), _multi_root(127, 3, 71),
               W.topk_tree(np.random.default_rng([2, 72]), 120, (16, 4, 2), 12),
               _multi_root(113, 2, 73), _multi_root(112, 1, 74), _multi_root(40, 2, 75)]
    paths = [chain_path(p, int(np.argmax(W.node_depths(p)))) for p in parents]
    w = custom(cfg, parents, paths, seed=128)
    state = rand_state(cfg, len(parents), seed=12)
    up = H.Uploaded(w)
    print(f"delta rule dense kernel sizes={[len(p) for p in parents]}", flush=True)
    got, err = H.run_verify(cfg, up, H.t_f32(state))
    assert err == 0
    assert H.slice_rel_err(got, o_verify(cfg, w, state), w.node_offsets) <= H.TOL
    st = H.t_f32(state)
    assert H.run_commit(cfg, up, st) == 0
    assert H.state_rel_err(st.cpu().numpy(), o_commit(cfg, w, state)) <= H.TOL


@pytest.mark.parametrize("hk, hv, cap", [(4, 8, 128), (4, 16, 128), (8, 16, 64)])
def test_delta_rule_dense_full_launch_ragged(hk, hv, cap):
    """The dense delta-rule kernel at the size of the benchmark's launch
    (B * Hv >= 2 x the GPU's compute units, so the grid runs in two rounds or
    more): group sizes 2 and 4, node caps 128 and 64, ragged multi-root trees
    of 1..cap nodes (full tiles among them), an empty request.  Every head of
    sampled requests against the oracle, verify and commit."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    B = -(-2 * cus // hv) + 3
    rng = np.random.default_rng([hk, hv, cap])
    sizes = [cap, cap - 1, 0, 1, 15, 16, 17] + [int(x) for x in rng.integers(1, cap + 1, B - 7)]
    parents = [_multi_root(T, 1 + b % 3, 900 + b) if T else np.zeros(0, np.int32)
               for b, T in enumerate(sizes)]
    paths = [chain_path(p, int(np.argmax(W.node_depths(p)))) if len(p) else [] for p in parents]
    cfg = cfg_of("gdn", batch=B, num_qk_heads=hk, num_v_heads=hv, d_k=128, d_v=128,
                 prefix_len=0, max_nodes=cap)
    w = custom(cfg, parents, paths, seed=hv)
    state = rand_state(cfg, B, seed=hk)
    up = H.Uploaded(w)
    keep = [0, 1, 3, 4, 5, 6, B // 2, B - 1]
    print(f"delta rule dense full launch: Hk={hk} Hv={hv} cap={cap} B={B} slots={B * hv} cus={cus} "
          f"sample={keep}", flush=True)
    got, err = H.run_verify(cfg, up, H.t_f32(state))
    assert err == 0
    ws = sub(w, keep)
    assert H.slice_rel_err(got[rows_of(w, keep)], o_verify(cfg, ws, state[keep]), ws.node_offsets) <= H.TOL
    st = H.t_f32(state)
    assert H.run_commit(cfg, up, st) == 0
    got_s = st.cpu().numpy()
    assert H.state_rel_err(got_s[keep], o_commit(cfg, ws, state[keep])) <= H.TOL
    np.testing.assert_array_equal(got_s[2], state[2])   # the empty request's slot


@pytest.mark.parametrize("max_nodes, trees", [
    (176, [("roots", 176, 1), ("roots", 100, 2), ("roots", 17, 3), ("topk", 64, 0)]),
    (256, [("roots", 256, 1), ("roots", 177, 3), ("roots", 90, 2), ("roots", 15, 1), ("topk", 200, 0)]),
])
def test_delta_rule_wide_cap_kernel(max_nodes, trees):
    """The delta rule's kernel for node caps beyond the tile walk's LDS (d =
    128, caps of 176..256): its level-by-level solve over branching,
    multi-root and partial-tile forests of several sizes in one batch (the
    wave topology serves trees of <= 64 nodes, the LDS one the others, and
    trees of < 16 nodes the vector path), verify and commit."""
    cfg = cfg_of("gdn", batch=len(trees), num_qk_heads=2, num_v_heads=4, d_k=128, d_v=128,
                 prefix_len=0, max_nodes=max_nodes)
    parents = []
    for k, (kind, T, roots) in enumerate(trees):
        if kind == "roots":
            parents.append(_multi_root(T, roots, 50 + k))
        else:
            parents.append(W.topk_tree(np.random.default_rng([k, 61]), T, (16, 4, 2), 12))
    paths = [chain_path(p, len(p) - 1) for p in parents]
    paths[1] = chain_path(parents[1], int(np.argmax(W.node_depths(parents[1]))))
    w = custom(cfg, parents, paths, seed=max_nodes)
    state = rand_state(cfg, len(trees), seed=11)
    up = H.Uploaded(w)
    print(f"delta rule wide cap max_nodes={max_nodes} sizes={[len(p) for p in parents]}", flush=True)
    got, err = H.run_verify(cfg, up, H.t_f32(state))
    assert err == 0
    assert H.slice_rel_err(got, o_verify(cfg, w, state), w.node_offsets) <= H.TOL
    st = H.t_f32(state)
    assert H.run_commit(cfg, up, st) == 0
    assert H.state_rel_err(st.cpu().numpy(), o_commit(cfg, w, state)) <= H.TOL


@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("max_nodes, sizes", [(80, [65, 80, 17]), (144, [144, 100, 70]), (256, [256, 129, 200])])
def test_tile_walk_gla_head_dims(d, max_nodes, sizes):
    """Gated linear attention over trees of more than 64 nodes (the tile-walk
    kernel) at every head dimension, for buckets of 80, 144 and 256 nodes
    (2 to 8 node chunks of 32) with ragged trees in one batch."""
    cfg = cfg_of("large", batch=len(sizes), num_qk_heads=2, num_v_heads=4, d_k=d, d_v=d,
                 prefix_len=0, max_nodes=max_nodes)
    parents = [_multi_root(T, 1, 10 + k) for k, T in enumerate(sizes)]
    paths = [chain_path(p, len(p) - 1) for p in parents]
    w = custom(cfg, parents, paths)
    state = rand_state(cfg, len(sizes))
    up = H.Uploaded(w)
    got, err = H.run_verify(cfg, up, H.t_f32(state))
    assert err == 0
    assert H.slice_rel_err(got, o_verify(cfg, w, state), w.node_offsets) <= H.TOL
    st = H.t_f32(state)
    assert H.run_commit(cfg, up, st) == 0
    assert H.state_rel_err(st.cpu().numpy(), o_commit(cfg, w, state)) <= H.TOL


@pytest.mark.parametrize("B", [3, 150, 260])
def test_delta_rule_commit_decay_extremes(B):
    """The delta-rule commit replays rows held as S divided by the running
    decay product and folds that product back into them whenever it leaves
    [2^-32, 2^32].  Three 45-step paths (two staging chunks) whose decays
    force folds within and across chunks: decays down to e^-8 per step; a
    zero decay (g = -inf) and an e^-50 one among decays of exactly one; and
    growing decays (g = +0.5).  The other requests commit short paths, and
    B (times 4 v-heads) puts the launch in each of its splits."""
    cfg = cfg_of("gdn", batch=B, num_qk_heads=2, num_v_heads=4, prefix_len=0, max_nodes=64)
    parents = [W.chain_tree(45)] * 3 + [W.chain_tree(3)] * (B - 3)
    paths = [list(range(45))] * 3 + [list(range(1 + b % 3)) for b in range(B - 3)]
    w = custom(cfg, parents, paths, seed=B)
    rng = np.random.default_rng([B, 17])
    g = w.g.copy()
    g[0:45] = -8.0 * rng.random((45, 4))
    g[45:90] = 0.0
    g[45 + 20] = -np.inf
    g[45 + 33] = -50.0
    g[90:135] = 0.5
    w = dataclasses.replace(w, g=g.astype(np.float32))
    state = rand_state(cfg, B, seed=B)
    up = H.Uploaded(w)
    print(f"delta-rule commit decay extremes B={B} slots={4 * B}", flush=True)
    st = H.t_f32(state)
    assert H.run_commit(cfg, up, st) == 0
    got = st.cpu().numpy()
    assert np.isfinite(got).all()
    assert H.state_rel_err(got, o_commit(cfg, w, state)) <= H.TOL


@pytest.mark.parametrize("name", ["large", "gdn"])
def test_deepest_tree_256_chain(name):
    cfg = cfg_of(name, batch=1, prefix_len=0, max_nodes=256)
    parent = W.chain_tree(256)
    w = custom(cfg, [parent], [list(range(256))])
    state = rand_state(cfg, 1, scale=0.1)
    up = H.Uploaded(w)
    got, err = H.run_verify(cfg, up, H.t_f32(state))
    assert err == 0
    assert H.slice_rel_err(got, o_verify(cfg, w, state), w.node_offsets) <= H.TOL
    st = H.t_f32(state)
    assert H.run_commit(cfg, up, st) == 0
    assert H.state_rel_err(st.cpu().numpy(), o_commit(cfg, w, state)) <= H.TOL


@pytest.mark.parametrize("name", ["production", "gdn", "large", "tiny"])
def test_query_scale(name):
    cfg = cfg_of(name, prefix_len=0, q_scale=0.0883883)
    w = W.make(cfg, requests=[0, 1])
    state = rand_state(cfg, 2)
    got, err = H.run_verify(cfg, H.Uploaded(w), H.t_f32(state))
    assert err == 0
    assert H.slice_rel_err(got, o_verify(cfg, w, state), w.node_offsets) <= H.TOL


# ----------------------------------------------------------------------------
# the full production batch, in the launch configuration bench.py times
# ----------------------------------------------------------------------------

def test_full_production_batch_sampled():
    """All 32 requests go through one launch of each kernel; the oracle
    checks sampled requests one by one (their S_pre from the oracle's own
    prefix recurrence; the other requests get random states)."""
    cfg = W.CONFIGS["production"]
    w = W.make(cfg)
    sample = [0, 13, 31]
    state = rand_state(cfg, cfg.batch, scale=0.5)
    state[sample] = H.oracle_prefix_state(cfg, 0, sample)
    up = H.Uploaded(w)
    got, err = H.run_verify(cfg, up, H.t_f32(state))
    assert err == 0
    assert np.isfinite(got).all()
    ws = sub(w, sample)
    e = H.slice_rel_err(got[rows_of(w, sample)], o_verify(cfg, ws, state[sample]), ws.node_offsets)
    print(f"full batch, sampled verify max slice rel err {e:.3e}")
    assert e <= H.TOL
    st = H.t_f32(state)
    assert H.run_commit(cfg, up, st) == 0
    e = H.state_rel_err(st.cpu().numpy()[sample], o_commit(cfg, ws, state[sample]))
    print(f"full batch, sampled commit max slot rel err {e:.3e}")
    assert e <= H.TOL
