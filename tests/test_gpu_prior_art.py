"""The prior-art prefix-sum pooling that bench.py --cumsum times beside the
forward (the paper's speed comparison) computes the same map: against the
oracle, with a bound that covers fp32 prefix sums over all kept points
(each cell's value is a difference of two prefixes, so its error scales with
the prefixes' size, not with the cell's)."""
import numpy as np
import pytest

import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("inner_scan", [False, True])
def test_prefix_sum_pooling_matches_oracle(oracle_lib, inner_scan):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2205_13542_amd as bp
    from bench import cumsum_trick_pool
    print("[prior art] nuscenes prefix-sum pooling", flush=True)
    w = wl.make("nuscenes", seed=9)
    plan = bp.Plan.from_rig(w.rig)
    _, sp, cs = plan.export()
    dev = torch.device("cuda:0")
    got = cumsum_trick_pool(torch.from_numpy(w.P).to(dev), torch.from_numpy(w.F).to(dev),
                            torch.from_numpy(sp.astype(np.int64)).to(dev),
                            torch.from_numpy(cs.astype(np.int64)).to(dev),
                            w.rig, w.channels, inner_scan=inner_scan).cpu().numpy()
    cop = oracle_lib.cell_map(w.rig)
    _, ref = oracle_lib.pool(w.rig, cop, w.P, w.F, want_f64=True)
    # size of the prefixes, in double, from the oracle's sums in cell order
    # (a running sum over the cells is the prefix over the sorted points at
    # the cells' ends); a parallel fp32 scan errs by about log2(K) roundings
    # of that size
    flat = ref.reshape(-1, w.channels)
    scale = np.abs(np.cumsum(flat, axis=0)).max(axis=0)[None, :]
    err = np.abs(got.reshape(-1, w.channels).astype(np.float64) - flat)
    bound = (4 * np.finfo(np.float32).eps * np.log2(max(int(cs[-1]), 2)) * scale
             + 1e-4 * np.sqrt(np.maximum(np.diff(cs), 1))[:, None])
    assert (err <= bound).all(), f"max err/bound {(err / bound).max():.3g}"
    plan.close()
