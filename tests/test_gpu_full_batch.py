"""Full batches of the gated-delta-rule workload (16 requests of 128-node
trees) and of the large-batch workload (128 requests of 16..256 nodes, one a
16-node chain) through one launch of each kernel, in the launch
configuration bench.py times (same problem, batch, node cap and grid), for
two steps: the second verifies new trees against the state the first
committed.  The fp64 oracle checks sampled requests one by one -- the first,
the last, the largest tree, and for the large workload the 16-node chain --
with S_pre from the oracle's own prefix recurrence; the other requests get
random states.  The production batch has the same test in test_gpu_edge."""
import numpy as np
import pytest

import oracle
from synth import workloads as W
from tests import gpu_helpers as H
from tests.test_gpu_edge import o_commit, o_verify, rand_state, rows_of, sub

pytestmark = pytest.mark.gpu


def _samples(name, w):
    sizes = np.diff(w.node_offsets)
    B = len(sizes)
    keep = {0, B // 2, B - 1, int(sizes.argmax())}
    if name == "large":
        chains = [b for b in range(B) if sizes[b] == 16 and
                  np.array_equal(w.parent[w.node_offsets[b]:w.node_offsets[b + 1]], W.chain_tree(16))]
        assert chains, "the large workload holds a 16-node chain"
        keep.add(chains[0])
    return sorted(keep)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name", ["gdn", "large"])
def test_full_batch_two_steps_sampled(name):
    cfg = W.CONFIGS[name]
    w0 = W.make(cfg, step=0)
    sample = _samples(name, w0)
    state = rand_state(cfg, cfg.batch, scale=0.5)
    state[sample] = H.oracle_prefix_state(cfg, 0, sample)
    st = H.t_f32(state)
    ref_state = state[sample].astype(np.float64)
    for step in range(2):
        w = w0 if step == 0 else W.make(cfg, step=step)
        up = H.Uploaded(w)
        print(f"{name} full batch step {step}: B={w.batch} N={w.N} sample={sample}", flush=True)
        got, err = H.run_verify(cfg, up, st)
        assert err == 0
        assert np.isfinite(got).all()
        ws = sub(w, sample)
        ref_o = o_verify(cfg, ws, ref_state)
        e = H.slice_rel_err(got[rows_of(w, sample)], ref_o, ws.node_offsets)
        print(f"  verify max slice rel err {e:.3e}", flush=True)
        assert e <= H.TOL
        assert H.run_commit(cfg, up, st) == 0
        ref_state = o_commit(cfg, ws, ref_state)
        got_s = st.cpu().numpy()
        assert np.isfinite(got_s).all()
        e = H.state_rel_err(got_s[sample], ref_state)
        print(f"  commit max slot rel err {e:.3e}", flush=True)
        assert e <= H.TOL
