"""Seeded input generators: determinism, tree shapes, bf16 rounding."""
import numpy as np
import pytest
import torch

from synth import workloads as W


def _depths(p):
    return W.node_depths(p)


def test_same_seed_same_bytes():
    a = W.make("production", seed=3, batch=4)
    b = W.make("production", seed=3, batch=4)
    c = W.make("production", seed=4, batch=4)
    for f in ("node_offsets", "parent", "q", "k", "v", "g", "path_offsets", "path"):
        assert getattr(a, f).tobytes() == getattr(b, f).tobytes()
    assert a.q.tobytes() != c.q.tobytes()
    # a request does not depend on which other requests are drawn
    d = W.make("production", seed=3, requests=[2])
    o = a.node_offsets
    assert d.q.tobytes() == a.q[o[2]:o[3]].tobytes()


@pytest.mark.parametrize("name", ["tiny", "mid", "production", "gdn"])
def test_tree_shapes(name):
    cfg = W.CONFIGS[name]
    w = W.make(name, batch=min(cfg.batch, 6))
    for b in range(w.batch):
        p = w.parent[w.node_offsets[b]:w.node_offsets[b + 1]]
        assert p[0] == -1 and np.all(p[1:] >= 0)
        assert np.all(p[1:] < np.arange(1, p.size))
        if cfg.tree[0] == "binary":
            np.testing.assert_array_equal(p, [-1, 0, 0, 1, 1, 2, 2, 3, 3, 4, 4, 5, 5, 6, 6])
        else:
            _, T, branching, cap = cfg.tree
            assert p.size == T
            d = _depths(p)
            assert d.max() <= cap
            # children per node never exceed the branching factor of its depth
            kids = np.bincount(p[1:], minlength=p.size)
            for i in range(p.size):
                nb = branching[d[i]] if d[i] < len(branching) else 1
                assert kids[i] <= nb
            # BFS order: depths are non-decreasing
            assert np.all(np.diff(d) >= 0)


def test_large_tree_mix():
    w = W.make("large", batch=8)
    sizes = np.diff(w.node_offsets)
    assert sizes[0] == 16 and sizes[1] == 256
    assert np.all((sizes[2:] >= 32) & (sizes[2:] <= 256))
    p0 = w.parent[:16]
    np.testing.assert_array_equal(p0, np.arange(-1, 15))
    for b in range(1, 8):
        p = w.parent[w.node_offsets[b]:w.node_offsets[b + 1]]
        assert np.all(p[1:] < np.arange(1, p.size)) and p[0] == -1
        assert _depths(p).max() <= 16


@pytest.mark.parametrize("name", ["tiny", "mid", "production", "gdn", "large"])
def test_paths_are_root_chains(name):
    cfg = W.CONFIGS[name]
    w = W.make(name, batch=min(cfg.batch, 5))
    for b in range(w.batch):
        p = w.parent[w.node_offsets[b]:w.node_offsets[b + 1]]
        path = w.path[w.path_offsets[b]:w.path_offsets[b + 1]]
        assert path.size >= 1
        prev = -1
        for a in path:
            assert p[a] == prev
            prev = a
        if cfg.path_rule[0] == "leaf":
            assert path.size == 4 and not np.any(p == path[-1])
        else:
            assert path.size <= cfg.path_rule[1]


def test_inputs_distributions():
    w = W.make("production", batch=2)
    n = np.linalg.norm(w.q.astype(np.float64), axis=-1)
    assert np.all(np.abs(n - 1) < 1e-2)
    # bf16 configs hold bf16-representable values
    assert np.all(W.round_bf16(w.v) == w.v)
    assert np.all(w.g < 0)
    t = W.make("tiny")
    assert t.q.dtype == np.float32 and np.any(W.round_bf16(t.v) != t.v)
    assert t.state.shape == (1, 1, 16, 16)


def test_bf16_rne_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(100000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 100000),
        np.array([0.0, -0.0, np.inf, -np.inf, 3.3895314e38, -3.3895314e38, 1e-45, -1e-45,
                  1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9], np.float32),
        # exact ties between two bf16 values: both even and odd neighbours
        (np.arange(1, 2000, dtype=np.uint32) << 16 | 0x8000).view(np.float32),
    ]).astype(np.float32)
    ours = W.bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    nan = np.array([np.nan, -np.nan], np.float32)
    assert np.all(np.isnan(W.bf16_to_f32(W.bf16_bits(nan))))


def test_prefix_chunks_independent():
    k0, v0, g0, b0 = W.prefix_chunk("gdn", 0, 3, 2)
    k1, v1, g1, b1 = W.prefix_chunk("gdn", 0, 3, 2)
    assert k0.tobytes() == k1.tobytes() and b0.tobytes() == b1.tobytes()
    assert k0.shape == (256, 16, 128) and v0.shape == (256, 32, 128)
    assert W.prefix_chunks("production") == 8 and W.prefix_chunks("mid") == 2
