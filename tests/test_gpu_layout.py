"""Channel-major copy of the BEV map (bevpool_to_nchw) on the GPU: bit-exact
against numpy's transpose of the same host array, on ragged tile counts,
strided rows and batches; and the pooled map in NCHW against the oracle's
map transposed by numpy."""
import ctypes

import numpy as np
import pytest

import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


@pytest.fixture(scope="module")
def pkg(torch_cuda):
    import paper_2205_13542_amd as pkg
    pkg._binding.load()
    return pkg


@pytest.mark.parametrize("B,ny,nx,C,ldi,off", [(2, 360, 360, 80, 80, 0), (1, 37, 29, 33, 33, 0),
                                               (3, 5, 7, 1, 1, 0), (1, 64, 64, 80, 96, 16),
                                               (2, 11, 13, 70, 75, 5), (1, 1, 1, 200, 200, 0),
                                               (1, 3, 50, 260, 260, 0), (2, 9, 9, 80, 96, 16)])
def test_to_nchw_matches_numpy_transpose(torch_cuda, pkg, B, ny, nx, C, ldi, off):
    print(f"[nchw] B={B} {ny}x{nx} C={C} ldi={ldi} off={off}", flush=True)
    torch = torch_cuda
    rng = np.random.default_rng(B * 1000 + C)
    host = rng.standard_normal((B, ny, nx, ldi)).astype(np.float32)
    x = torch.from_numpy(host).cuda()
    out = torch.full((B, C, ny, nx), float("nan"), device="cuda")
    pkg.to_nchw(x[..., off:off + C], out=out)
    torch.cuda.synchronize()
    ref = np.ascontiguousarray(np.transpose(host[..., off:off + C], (0, 3, 1, 2)))
    assert np.array_equal(out.cpu().numpy(), ref)


def test_pooled_map_in_nchw(torch_cuda, pkg, oracle_lib):
    torch = torch_cuda
    w = wl.make("nuscenes_tilted", seed=3)
    plan = pkg.Plan.from_rig(w.rig)
    P = torch.from_numpy(w.P).cuda()
    F = torch.from_numpy(w.F).cuda()
    got = pkg.to_nchw(plan.forward(P, F)).cpu().numpy()
    cop = oracle_lib.cell_map(w.rig)
    _, ref = oracle_lib.pool(w.rig, cop, w.P, w.F, want_f64=True)
    n = np.bincount(cop[cop >= 0], minlength=w.rig.n_cells).reshape(w.rig.ny, w.rig.nx)
    err = np.abs(got.astype(np.float64) - np.transpose(ref, (0, 3, 1, 2)))
    assert (err <= 1e-4 * np.sqrt(np.maximum(n, 1))[None, None]).all()
    plan.close()


def test_to_nchw_argument_errors(torch_cuda, pkg):
    torch = torch_cuda
    lib = pkg._binding.load()
    x = torch.zeros((1, 4, 4, 8), device="cuda")
    y = torch.zeros((1, 8, 4, 4), device="cuda")
    vp = ctypes.c_void_p
    bad = pkg._binding.BEVPOOL_ERR_INVALID_ARG
    assert lib.bevpool_to_nchw(None, 8, vp(y.data_ptr()), 1, 4, 4, 8, None) == bad
    assert lib.bevpool_to_nchw(vp(x.data_ptr()), 7, vp(y.data_ptr()), 1, 4, 4, 8, None) == bad
    assert lib.bevpool_to_nchw(vp(x.data_ptr()), 8, vp(y.data_ptr()), 0, 4, 4, 8, None) == bad
    assert lib.bevpool_to_nchw(vp(x.data_ptr()), 1 << 31, vp(y.data_ptr()), 1, 4, 4, 8,
                               None) == pkg._binding.BEVPOOL_ERR_OVERFLOW
    assert lib.bevpool_to_nchw(vp(x.data_ptr()), 8, vp(y.data_ptr()), 1, 4, 4, 8, None) == 0
    torch.cuda.synchronize()
