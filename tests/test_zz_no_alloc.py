"""The association entry point that allocates nothing (bevpool_associate_noalloc)
against the allocating one (bevpool_plan, then bevpool_plan_export): two calls
in a row on one device, the second with a smaller rig, each bit-exact; the
sizes beyond its limits are refused."""
import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import workloads as wl  # noqa: E402


@pytest.fixture(scope="module")
def torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _reference(pkg, rig):
    plan = pkg.Plan.from_rig(rig)
    cop, sp, cs = plan.export()
    plan.close()
    return cop, sp, cs


@pytest.mark.gpu
def test_associate_noalloc_matches_plan_twice(torch_cuda):
    import paper_2205_13542_amd as pkg
    torch = torch_cuda
    free_before = None
    for name in ("nuscenes", "tiny"):       # the second call is smaller
        rig = wl.make(name, seed=0).rig
        print(f"[no-alloc] {name}: {rig.n_points} points, {rig.n_cells} cells", flush=True)
        cop_ref, sp_ref, cs_ref = _reference(pkg, rig)
        cop = torch.full((rig.n_points,), -7, dtype=torch.int32, device="cuda")
        sp = torch.full((rig.n_points,), -7, dtype=torch.int32, device="cuda")
        cs = torch.full((rig.n_cells + 1,), -7, dtype=torch.int32, device="cuda")
        torch.cuda.synchronize()
        free0 = torch.cuda.mem_get_info()[0]
        pkg.associate_noalloc(rig, cop, sp, cs)
        torch.cuda.synchronize()
        free1 = torch.cuda.mem_get_info()[0]
        if free_before is not None:          # past the first call (module load)
            assert free1 == free0, "the call changed the device's free memory"
        free_before = free1
        cop_h, sp_h, cs_h = cop.cpu().numpy(), sp.cpu().numpy(), cs.cpu().numpy()
        assert np.array_equal(cop_h, cop_ref)
        assert np.array_equal(cs_h, cs_ref)
        kept = int(cs_ref[-1])
        assert np.array_equal(sp_h[:kept], sp_ref[:kept])
        assert np.array_equal(sp_h[kept:], np.flatnonzero(cop_ref < 0).astype(np.int32))


@pytest.mark.gpu
def test_associate_noalloc_refuses_sizes_beyond_its_limits(torch_cuda):
    import paper_2205_13542_amd as pkg
    torch = torch_cuda
    rig = wl.make("highres", seed=0).rig          # 16 M points, above 2^22
    cop = torch.empty((rig.n_points,), dtype=torch.int32, device="cuda")
    sp = torch.empty((rig.n_points,), dtype=torch.int32, device="cuda")
    cs = torch.empty((rig.n_cells + 1,), dtype=torch.int32, device="cuda")
    with pytest.raises(pkg.BevpoolError, match="no-allocation maximum"):
        pkg.associate_noalloc(rig, cop, sp, cs)
