"""Verification against the oracle with the library built with -DTL_DEBUG
(libtreelin_debug.so): every verify kernel fills its LDS with NaN before
first use.  Where a kernel reads LDS it has not written -- the rows past a
tree's last node in the small-tree kernel, which by design only meet
coefficients that the ancestor mask selects to zero, the tile walk's
padding, the delta rule's zeroed U columns -- a NaN would reach the outputs.
So parity here shows that every such read is either written first or
discarded by a select, across the kernels: the small-tree kernel at tree
sizes that leave rows past T in each 16-node tile and 32-node chunk, the tile
walk for both rules, the delta rule's wide-cap kernel and the vector path."""
import os

import numpy as np
import pytest

from synth import workloads as W
from tests import gpu_helpers as H
from tests.test_gpu_edge import _multi_root, cfg_of, chain_path, custom, o_verify, rand_state
from tests.test_gpu_parity import PARITY_CASES, _oracle_verify, _workload
from paper_2608_01651_amd import treelin as tl

pytestmark = pytest.mark.gpu

DEBUG_LIB = os.path.join(os.path.dirname(tl._LIB_PATH), "libtreelin_debug.so")


@pytest.fixture(scope="module", autouse=True)
def debug_library():
    if not os.path.exists(DEBUG_LIB):
        raise RuntimeError(f"{DEBUG_LIB} is missing: build it with `python -m paper_2608_01651_amd.build`")
    saved = (tl._lib, tl._LIB_PATH)
    tl._lib, tl._LIB_PATH = None, DEBUG_LIB
    tl.lib()
    yield
    tl._lib, tl._LIB_PATH = saved


@pytest.mark.parametrize("name", list(PARITY_CASES))
def test_poisoned_lds_workloads(name):
    cfg, w, state = _workload(name)
    got, err = H.run_verify(cfg, H.Uploaded(w), H.t_f32(state))
    assert err == 0
    assert np.isfinite(got).all()
    e = H.slice_rel_err(got, _oracle_verify(cfg, w, state), w.node_offsets)
    print(f"{name}: poisoned-LDS verify max slice rel err {e:.3e}", flush=True)
    assert e <= H.TOL


@pytest.mark.parametrize("base, mode, max_nodes, sizes", [
    ("production", W.GLA, 64, [16, 17, 31, 33, 50, 63, 64, 15, 1]),    # small-tree kernel
    ("mid", W.GLA, 64, [20, 47]),                                       # one v-head per block
    ("large", W.GLA, 256, [65, 80, 129, 200, 256, 7]),                  # tile walk, gated linear attention
    ("gdn", W.GDN, 128, [128, 65, 100, 17, 3]),                         # tile walk, delta rule
    ("gdn", W.GDN, 256, [256, 177, 90, 40, 12]),                        # the delta rule's wide-cap kernel
])
def test_poisoned_lds_ragged_trees(base, mode, max_nodes, sizes):
    cfg = cfg_of(base, batch=len(sizes), mode=mode, prefix_len=0, max_nodes=max_nodes,
                 num_qk_heads=2, num_v_heads=4 if base != "mid" else 2)
    parents = [_multi_root(T, 1 + (k % 3) if T > 3 else 1, 70 + k) for k, T in enumerate(sizes)]
    paths = [chain_path(p, len(p) - 1) for p in parents]
    w = custom(cfg, parents, paths, seed=max_nodes + len(sizes))
    state = rand_state(cfg, len(sizes), seed=3)
    got, err = H.run_verify(cfg, H.Uploaded(w), H.t_f32(state))
    assert err == 0
    assert np.isfinite(got).all()
    assert H.slice_rel_err(got, o_verify(cfg, w, state), w.node_offsets) <= H.TOL
