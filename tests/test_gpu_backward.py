"""Backward pass on the GPU against the oracle's gradients (same inputs, same
association). Bounds, per element: |dP - ref| <= 1e-4 sqrt(C) (a dot product
of C terms of order one) and |dF - ref| <= 1e-4 sqrt(k), k the pixel's kept
depth bins; dropped points and pixels without kept points exactly 0."""
import dataclasses

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
def pkg():
    import paper_2205_13542_amd as bp
    bp._binding.load()
    return bp


def _say(msg):
    print(msg, flush=True)


def _dev(torch, a, dtype):
    t = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return t.to({"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[dtype]).contiguous()


def _host_values(torch, a, dtype):
    """The values the GPU sees: a rounded to dtype, widened back to fp32."""
    return _dev(torch, a, dtype).float().cpu().numpy()


def _check(torch, pkg, oracle_lib, w, G, dtype="f32", want_depth=True, want_feat=True):
    rig = w.rig
    P = _dev(torch, w.P, dtype)
    F = _dev(torch, w.F, dtype)
    Gd = torch.from_numpy(G).cuda().contiguous()
    plan = pkg.Plan.from_rig(rig)
    gd, gf = plan.backward(Gd, P, F, want_depth=want_depth, want_feat=want_feat)
    torch.cuda.synchronize()
    cop = oracle_lib.cell_map(rig)
    refP, refF = oracle_lib.backward(rig, cop, _host_values(torch, w.P, dtype),
                                     _host_values(torch, w.F, dtype), G)
    C = w.channels
    kept = cop >= 0
    if want_depth:
        got = gd.cpu().numpy().reshape(w.batch, -1)
        ref = refP.reshape(w.batch, -1)
        err = np.abs(got.astype(np.float64) - ref)
        assert (err <= 1e-4 * np.sqrt(C)).all(), f"dP max err {err.max():.3g}"
        assert (got[:, ~kept] == 0).all()
    else:
        assert gd is None
    if want_feat:
        got = gf.cpu().numpy().reshape(w.batch, rig.n_pixels, C)
        ref = refF.reshape(w.batch, rig.n_pixels, C)
        k = kept.reshape(rig.n_cams, rig.n_depth, -1).sum(axis=1).reshape(-1)
        bound = 1e-4 * np.sqrt(np.maximum(k, 1))[None, :, None]
        err = np.abs(got.astype(np.float64) - ref)
        assert (err <= bound).all(), f"dF max err/bound {(err / bound).max():.3g}"
        assert (got[:, k == 0] == 0).all()
    else:
        assert gf is None
    plan.close()
    return gd, gf


def _grad(w, seed):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((w.batch, w.rig.ny, w.rig.nx, w.channels)).astype(np.float32)


@pytest.mark.parametrize("name,seed", [("tiny", 0), ("tiny_identity", 1), ("nuscenes", 2),
                                       ("nuscenes_tilted", 3), ("nuscenes_tilt1", 5)])
def test_backward_matches_oracle(torch_cuda, pkg, oracle_lib, name, seed):
    """Level rig: every combo clean (one gradient row per combo); tilted rig:
    mostly rows with cells of their own."""
    _say(f"[backward] {name} seed={seed}")
    w = wl.make(name, seed=seed)
    _check(torch_cuda, pkg, oracle_lib, w, _grad(w, seed + 10))


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_backward_reduced_precision_inputs(torch_cuda, pkg, oracle_lib, dtype):
    _say(f"[backward] nuscenes {dtype}")
    w = wl.make("nuscenes", seed=4)
    _check(torch_cuda, pkg, oracle_lib, w, _grad(w, 14), dtype=dtype)


@pytest.mark.parametrize("channels", [1, 5, 17, 64, 81, 160, 260])
def test_backward_channel_counts(torch_cuda, pkg, oracle_lib, channels):
    """Every lane-chunk count, 4-element lanes (160), and channel slices
    (81, 160, 260: dP adds the slices' dot products)."""
    _say(f"[backward] nuscenes_tilted C={channels}")
    w = wl.make("nuscenes_tilted", seed=5, channels=channels)
    _check(torch_cuda, pkg, oracle_lib, w, _grad(w, channels))


def test_backward_batch_and_single_outputs(torch_cuda, pkg, oracle_lib):
    _say("[backward] batch 2, one output at a time")
    w = wl.make("nuscenes", seed=6, batch=2)
    G = _grad(w, 16)
    gd, gf = _check(torch_cuda, pkg, oracle_lib, w, G)
    gd1, _ = _check(torch_cuda, pkg, oracle_lib, w, G, want_feat=False)
    _, gf1 = _check(torch_cuda, pkg, oracle_lib, w, G, want_depth=False)
    assert torch_cuda.equal(gd, gd1) and torch_cuda.equal(gf, gf1)


def test_backward_deterministic(torch_cuda, pkg):
    torch = torch_cuda
    w = wl.make("nuscenes_tilted", seed=7)
    plan = pkg.Plan.from_rig(w.rig)
    P, F = _dev(torch, w.P, "f32"), _dev(torch, w.F, "f32")
    G = torch.from_numpy(_grad(w, 17)).cuda()
    a = plan.backward(G, P, F)
    b = plan.backward(G, P, F)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
    plan.close()


def test_backward_adjoint_on_gpu(torch_cuda, pkg):
    """<G, forward(P, F)> = <P, dP> = <F, dF> with the GPU's own forward and
    backward, in double on the host."""
    torch = torch_cuda
    w = wl.make("nuscenes", seed=8)
    plan = pkg.Plan.from_rig(w.rig)
    P, F = _dev(torch, w.P, "f32"), _dev(torch, w.F, "f32")
    G = torch.from_numpy(_grad(w, 18)).cuda()
    out = plan.forward(P, F)
    gd, gf = plan.backward(G, P, F)
    torch.cuda.synchronize()
    d = lambda x: x.double().cpu()
    lhs = float((d(G) * d(out)).sum())
    via_p = float((d(P) * d(gd)).sum())
    via_f = float((d(F) * d(gf)).sum())
    scale = float((d(G).abs() * d(out).abs()).sum())
    assert abs(lhs - via_p) <= 1e-5 * scale and abs(lhs - via_f) <= 1e-5 * scale
    plan.close()


def test_autograd_function_matches_oracle(torch_cuda, pkg, oracle_lib):
    """bev_pool under autograd: a scalar loss sum(out * G) gives the oracle's
    gradients for G (and the same tensors as calling backward directly)."""
    torch = torch_cuda
    w = wl.make("nuscenes_tilted", seed=19)
    plan = pkg.Plan.from_rig(w.rig)
    P = torch.from_numpy(w.P).cuda().requires_grad_(True)
    F = torch.from_numpy(w.F).cuda().requires_grad_(True)
    G = torch.from_numpy(_grad(w, 29)).cuda()
    out = pkg.bev_pool(P, F, plan)
    (out * G).sum().backward()
    torch.cuda.synchronize()
    gd, gf = plan.backward(G, P.detach(), F.detach())
    assert torch.equal(P.grad, gd) and torch.equal(F.grad, gf)
    cop = oracle_lib.cell_map(w.rig)
    refP, refF = oracle_lib.backward(w.rig, cop, w.P, w.F, _grad(w, 29))
    assert (np.abs(P.grad.cpu().numpy().astype(np.float64) - refP) <= 1e-4 * np.sqrt(w.channels)).all()
    k = (cop >= 0).reshape(w.rig.n_cams, w.rig.n_depth, -1).sum(axis=1).reshape(-1)
    bound = 1e-4 * np.sqrt(np.maximum(k, 1))[None, :, None]
    got = F.grad.cpu().numpy().reshape(w.batch, w.rig.n_pixels, w.channels)
    assert (np.abs(got - refF.reshape(got.shape)) <= bound).all()
    plan.close()


# ------------------------------------------------------------ matrix-core path
#
# Level rigs send every block to the matrix-core kernel when the channel count
# is a multiple of 4 and the rows are aligned; otherwise, and for blocks with a
# combo that is not clean, the per-row kernel runs.

from test_gpu_parity import RIGS  # noqa: E402


def _rig_workload(rig, channels, seed, batch=1, dtype="f32"):
    P, F = wl.frames(rig, channels, batch, "peaked", seed=seed, dtype=dtype)
    return wl.Workload("c", rig, channels, batch, dtype, P, F)


@pytest.mark.parametrize("channels", [4, 16, 48, 64, 80, 84, 160, 200, 5, 17, 81])
def test_backward_level_channel_counts(torch_cuda, pkg, oracle_lib, channels):
    """Matrix-core launches of 1..5 channel tiles, a ragged last tile (84,
    200: slices of 80 then 4 or 40), several slices adding into dP (160,
    200); 5, 17 and 81 channels take the per-row kernel."""
    _say(f"[backward level] nuscenes C={channels}")
    w = _rig_workload(wl.ring_rig(), channels, seed=channels)
    _check(torch_cuda, pkg, oracle_lib, w, _grad(w, channels + 1))


@pytest.mark.parametrize("name", ["odd", "odd_tilted", "anisotropic", "coarse", "coarse_tilted",
                                  "one_cell", "empty", "tiny_identity", "tall"])
@pytest.mark.parametrize("channels", [8, 20])
def test_backward_edge_rigs(torch_cuda, pkg, oracle_lib, name, channels):
    """Odd sizes (27 columns: the last column pair has one column; 13 rows: a
    partial row block; 37 bins: partial depth steps), an empty grid, one
    cell, cells fed by many combos, and 16,400 rows (no clean combo)."""
    _say(f"[backward edge] {name} C={channels}")
    w = _rig_workload(RIGS[name](), channels, seed=channels + 3)
    _check(torch_cuda, pkg, oracle_lib, w, _grad(w, channels + 7))


def _one_tilted_camera_rig():
    """The ring rig with camera 0 pitched 5 degrees: its blocks hold combos
    that are not clean, the other cameras' blocks are all clean."""
    base = wl.ring_rig()
    tilted = wl.tilt_rig(base, 5.0, 2.0)
    E = base.extrinsics.copy()
    E[0] = tilted.extrinsics[0]
    return dataclasses.replace(base, extrinsics=E)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_backward_mixed_blocks(torch_cuda, pkg, oracle_lib, dtype):
    """One call runs both kernels on disjoint blocks."""
    _say(f"[backward mixed] one tilted camera {dtype}")
    w = _rig_workload(_one_tilted_camera_rig(), 80, seed=21, batch=2, dtype=dtype)
    _check(torch_cuda, pkg, oracle_lib, w, _grad(w, 22), dtype=dtype)


def test_backward_highres(torch_cuda, pkg, oracle_lib):
    """6 x 236 bins x 64 x 176, C = 128 (slices of 80 and 48 channels)."""
    _say("[backward highres] C=128")
    w = wl.make("highres", seed=3)
    _check(torch_cuda, pkg, oracle_lib, w, _grad(w, 23))


def test_backward_unaligned_features(torch_cuda, pkg, oracle_lib):
    """F one element past a 16-byte boundary: the per-row kernel takes every
    block; the result matches the aligned call within the bounds."""
    torch = torch_cuda
    _say("[backward] unaligned F")
    w = _rig_workload(wl.ring_rig(), 80, seed=24)
    plan = pkg.Plan.from_rig(w.rig)
    P = _dev(torch, w.P, "f32")
    buf = torch.empty(w.F.size + 1, dtype=torch.float32, device="cuda")
    buf[1:] = torch.from_numpy(w.F.reshape(-1)).cuda()
    F_un = buf[1:].view(w.F.shape)
    G = torch.from_numpy(_grad(w, 25)).cuda()
    gd, gf = plan.backward(G, P, F_un)
    torch.cuda.synchronize()
    cop = oracle_lib.cell_map(w.rig)
    refP, refF = oracle_lib.backward(w.rig, cop, w.P, w.F, _grad(w, 25))
    assert (np.abs(gd.cpu().numpy().astype(np.float64) - refP) <= 1e-4 * np.sqrt(80)).all()
    k = (cop >= 0).reshape(w.rig.n_cams, w.rig.n_depth, -1).sum(axis=1).reshape(-1)
    bound = 1e-4 * np.sqrt(np.maximum(k, 1))[None, :, None]
    got = gf.cpu().numpy().reshape(1, w.rig.n_pixels, 80)
    assert (np.abs(got - refF.reshape(got.shape)) <= bound).all()
    plan.close()


def test_backward_level_deterministic(torch_cuda, pkg):
    torch = torch_cuda
    w = wl.make("nuscenes", seed=26)
    plan = pkg.Plan.from_rig(w.rig)
    P, F = _dev(torch, w.P, "f32"), _dev(torch, w.F, "f32")
    G = torch.from_numpy(_grad(w, 27)).cuda()
    a = plan.backward(G, P, F)
    b = plan.backward(G, P, F)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
    plan.close()
