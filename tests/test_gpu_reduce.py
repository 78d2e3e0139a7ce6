"""Mean and max pooling, strided outputs and z slabs on the GPU (through the
C ABI's bevpool_forward_ex) against the oracle, on the same seeded inputs.

Bounds, per element:
- max: equal in value to the oracle's max, which is exact in double and
  rounded once to fp32. Both sides see the same products: a float times a
  float (or a widened bf16/fp16 value) rounded once, and rounding is
  monotonic, so the largest rounded product is the rounded largest product.
- mean: |gpu - ref| <= 1e-4 / sqrt(n) + 1e-6 |ref| with n the cell's point
  count: the sum's bound 1e-4 sqrt(n) divided by n, plus the rounding of the
  division.
- sum into a strided map: the forward's bound, 1e-4 sqrt(n).
Cells without points are exactly 0 in every mode; floats of the map outside
the written channels keep their previous contents.
"""
import dataclasses
import sys

import numpy as np
import pytest

import workloads as wl

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


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


def _coarse(rig):
    return dataclasses.replace(rig, nx=36, ny=36, cell_x=3.0, cell_y=3.0)


RIGS = {
    "tiny": wl.tiny_rig,
    "nuscenes": wl.ring_rig,                                   # column items + combine
    "nuscenes_tilted": lambda: wl.tilt_rig(wl.ring_rig()),     # generic cells, light and heavy
    "nuscenes_tilt1": lambda: wl.tilt_rig(wl.ring_rig(), 1.0, 0.5),   # row segments, several passes
    "coarse": lambda: _coarse(wl.ring_rig()),                  # many slots per cell
    "coarse_tilted": lambda: _coarse(wl.tilt_rig(wl.ring_rig())),
    "empty": lambda: dataclasses.replace(wl.tiny_rig(), x_min=100.0),
}

_TDT = {"f32": "float32", "bf16": "bfloat16", "f16": "float16"}


def _inputs(torch, rig, C, seed, dtype="f32", batch=1):
    P, F = wl.frames(rig, C, batch, "peaked", seed=seed, dtype=dtype)
    dt = getattr(torch, _TDT[dtype])
    Pd = torch.from_numpy(P).cuda().to(dt).contiguous()
    Fd = torch.from_numpy(F).cuda().to(dt).contiguous()
    # the values the GPU reads, widened exactly to fp32
    return Pd, Fd, Pd.float().cpu().numpy(), Fd.float().cpu().numpy()


def _counts(oracle_lib, rig, cop):
    return np.bincount(cop[cop >= 0], minlength=rig.n_cells).reshape(rig.ny, rig.nx)


def _check_reduce(got, ref, n, mode):
    """got fp32 [B][ny][nx][C], ref float64, n int [ny][nx]."""
    n4 = n[None, :, :, None]
    if mode == "max":
        assert np.array_equal(got, ref.astype(np.float32)), \
            f"max: {np.sum(got != ref.astype(np.float32))} elements differ"
    else:
        bound = 1e-4 / np.sqrt(np.maximum(n4, 1)) + 1e-6 * np.abs(ref)
        err = np.abs(got.astype(np.float64) - ref)
        assert (err <= bound).all(), f"mean: max err/bound {(err / bound).max():.3g}"
    assert (got[:, n == 0] == 0).all()


@pytest.mark.parametrize("mode", ["mean", "max"])
@pytest.mark.parametrize("name,C", [("tiny", 8), ("nuscenes", 80), ("nuscenes_tilted", 80),
                                    ("nuscenes_tilt1", 80), ("coarse", 16), ("coarse_tilted", 16),
                                    ("empty", 8)])
def test_reduce_matches_oracle(torch_cuda, pkg, oracle_lib, name, C, mode):
    _say(f"[reduce] {name} C={C} {mode}")
    torch = torch_cuda
    rig = RIGS[name]()
    Pd, Fd, Ph, Fh = _inputs(torch, rig, C, seed=11)
    plan = pkg.Plan.from_rig(rig)
    out = torch.full((1, rig.ny, rig.nx, C), float("nan"), device="cuda")
    plan.forward(Pd, Fd, out=out, reduce=mode)
    torch.cuda.synchronize()
    cop = oracle_lib.cell_map(rig)
    ref = oracle_lib.pool_reduce(rig, cop, Ph, Fh, mode)
    _check_reduce(out.cpu().numpy(), ref, _counts(oracle_lib, rig, cop), mode)
    plan.close()


@pytest.mark.parametrize("mode", ["mean", "max"])
@pytest.mark.parametrize("C", [1, 5, 17, 64, 81, 128, 160])
def test_reduce_channel_counts(torch_cuda, pkg, oracle_lib, C, mode):
    """Every lane-chunk count, channel slices (81, 128, 160), and 64-channel
    slices moved as 16-byte lanes (64, 128)."""
    _say(f"[reduce] nuscenes_tilted C={C} {mode}")
    torch = torch_cuda
    rig = RIGS["nuscenes_tilted"]()
    Pd, Fd, Ph, Fh = _inputs(torch, rig, C, seed=C)
    plan = pkg.Plan.from_rig(rig)
    out = plan.forward(Pd, Fd, reduce=mode)
    torch.cuda.synchronize()
    cop = oracle_lib.cell_map(rig)
    ref = oracle_lib.pool_reduce(rig, cop, Ph, Fh, mode)
    _check_reduce(out.cpu().numpy(), ref, _counts(oracle_lib, rig, cop), mode)
    plan.close()


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_reduce_reduced_precision_batch(torch_cuda, pkg, oracle_lib, dtype):
    """bf16 / fp16 inputs, two frames in one call, both modes."""
    _say(f"[reduce] nuscenes {dtype} batch 2")
    torch = torch_cuda
    rig = RIGS["nuscenes"]()
    Pd, Fd, Ph, Fh = _inputs(torch, rig, 80, seed=21, dtype=dtype, batch=2)
    plan = pkg.Plan.from_rig(rig)
    cop = oracle_lib.cell_map(rig)
    n = _counts(oracle_lib, rig, cop)
    for mode in ("mean", "max"):
        out = plan.forward(Pd, Fd, reduce=mode)
        torch.cuda.synchronize()
        _check_reduce(out.cpu().numpy(), oracle_lib.pool_reduce(rig, cop, Ph, Fh, mode), n, mode)
    plan.close()


def test_reduce_deterministic_and_sum_unchanged(torch_cuda, pkg):
    """Repeated mean/max calls are bitwise equal; reduce="sum" through
    bevpool_forward_ex equals bevpool_forward bitwise."""
    torch = torch_cuda
    rig = RIGS["nuscenes_tilted"]()
    Pd, Fd, _, _ = _inputs(torch, rig, 80, seed=31)
    plan = pkg.Plan.from_rig(rig)
    for mode in ("mean", "max"):
        a = plan.forward(Pd, Fd, reduce=mode)
        b = plan.forward(Pd, Fd, reduce=mode)
        assert torch.equal(a, b)
    s0 = plan.forward(Pd, Fd)
    s1 = torch.empty_like(s0)
    pkg.bevpool_forward_ex(Pd.data_ptr(), Fd.data_ptr(), plan.handle, s1.data_ptr(), 80, 1, 80,
                           pkg.BEVPOOL_F32, pkg.BEVPOOL_SUM,
                           torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert torch.equal(s0, s1)
    plan.close()


@pytest.mark.parametrize("name,C,ldo,off", [("nuscenes", 80, 96, 16), ("nuscenes", 80, 83, 3),
                                            ("nuscenes_tilted", 80, 160, 80),
                                            ("coarse", 16, 40, 24), ("nuscenes_tilted", 81, 90, 9)])
def test_strided_output(torch_cuda, pkg, oracle_lib, name, C, ldo, off):
    """Sum into channels [off, off + C) of rows ldo floats apart (aligned and
    unaligned strides); the other floats of the map keep their sentinel."""
    _say(f"[strided] {name} C={C} ldo={ldo} off={off}")
    torch = torch_cuda
    rig = RIGS[name]()
    Pd, Fd, Ph, Fh = _inputs(torch, rig, C, seed=41, batch=2)
    plan = pkg.Plan.from_rig(rig)
    big = torch.full((2, rig.ny, rig.nx, ldo), -7.0, device="cuda")
    plan.forward(Pd, Fd, out=big[..., off:off + C])
    torch.cuda.synchronize()
    got = big.cpu().numpy()
    cop = oracle_lib.cell_map(rig)
    _, ref = oracle_lib.pool(rig, cop, Ph, Fh, want_f64=True)
    n = _counts(oracle_lib, rig, cop)[None, :, :, None]
    err = np.abs(got[..., off:off + C].astype(np.float64) - ref)
    assert (err <= 1e-4 * np.sqrt(np.maximum(n, 1))).all()
    assert (got[..., :off] == -7.0).all() and (got[..., off + C:] == -7.0).all()
    plan.close()


@pytest.mark.parametrize("name", ["nuscenes", "nuscenes_tilted"])
@pytest.mark.parametrize("mode", ["sum", "mean", "max"])
def test_z_slabs(torch_cuda, pkg, oracle_lib, name, mode):
    """Four 4 m slabs from z = -8 m, flattened by channel concatenation,
    against the oracle's per-slab pooling."""
    _say(f"[slabs] {name} {mode}")
    torch = torch_cuda
    rig = dataclasses.replace(RIGS[name](), z_min=-8.0, z_cell=4.0)
    C, nz = 16, 4
    Pd, Fd, Ph, Fh = _inputs(torch, rig, C, seed=51)
    sp = pkg.SlabPlan.from_rig(rig, nz)
    got = sp.forward(Pd, Fd, reduce=mode).cpu().numpy()
    ref = oracle_lib.pool_slabs(rig, nz, Ph, Fh, mode)
    cop = oracle_lib.cell_map(rig, nz)
    counts = np.bincount(cop[cop >= 0], minlength=rig.n_cells * nz).reshape(rig.ny, rig.nx, nz)
    for iz in range(nz):
        n = counts[..., iz]
        g = got[..., iz * C:(iz + 1) * C]
        e = ref[..., iz * C:(iz + 1) * C]
        if mode == "sum":
            n4 = n[None, :, :, None]
            assert (np.abs(g.astype(np.float64) - e) <= 1e-4 * np.sqrt(np.maximum(n4, 1))).all()
            assert (g[:, n == 0] == 0).all()
        else:
            _check_reduce(g, e, n, mode)
        assert n.sum() > 0
    sp.close()


def test_reduce_argument_errors(torch_cuda, pkg):
    torch = torch_cuda
    rig = RIGS["tiny"]()
    Pd, Fd, _, _ = _inputs(torch, rig, 8, seed=61)
    plan = pkg.Plan.from_rig(rig)
    out = torch.empty((1, rig.ny, rig.nx, 8), device="cuda")
    lib = pkg._binding.load()
    import ctypes
    vp = ctypes.c_void_p
    s = torch.cuda.current_stream().cuda_stream
    args = (vp(Pd.data_ptr()), vp(Fd.data_ptr()), vp(plan.handle), vp(out.data_ptr()))
    assert lib.bevpool_forward_ex(*args, 7, 1, 8, 0, 0, vp(s)) == pkg._binding.BEVPOOL_ERR_INVALID_ARG
    assert lib.bevpool_forward_ex(*args, 8, 1, 8, 0, 3, vp(s)) == pkg._binding.BEVPOOL_ERR_INVALID_ARG
    assert lib.bevpool_forward_ex(*args, 8, 1, 8, 0, -1, vp(s)) == pkg._binding.BEVPOOL_ERR_INVALID_ARG
    assert lib.bevpool_forward_ex(*args, 1 << 40, 1, 8, 0, 0, vp(s)) == pkg._binding.BEVPOOL_ERR_OVERFLOW
    assert lib.bevpool_forward_ex(*args, 8, 1, 8, 0, 2, vp(s)) == 0
    with pytest.raises(pkg.BevpoolError):
        plan.forward(Pd, Fd, reduce="median")
    with pytest.raises(pkg.BevpoolError):
        plan.forward(Pd, Fd, reduce="max", events=(torch.cuda.Event(enable_timing=True),
                                                   torch.cuda.Event(enable_timing=True)))
    torch.cuda.synchronize()
    plan.close()


@pytest.mark.parametrize("name,nz", [("nuscenes", 4), ("nuscenes_tilted", 3), ("tiny", 2)])
def test_slab_plan_bit_exact(pkg, oracle_lib, name, nz):
    """One plan over nz stacked slabs (bevpool_plan_slabs): cell map, sorted
    points and interval table equal to the oracle's bit for bit, and every
    cell with points is served by columns or gathered."""
    _say(f"[slab plan] {name} nz={nz}")
    base = RIGS[name]()
    rig = dataclasses.replace(base, z_cell=base.z_cell / nz)
    plan = pkg.SlabPlan.from_rig(rig, nz)
    cop, sp, cs = plan.export()
    rcop, rsp, rcs = oracle_lib.plan_slabs(rig, nz)
    assert np.array_equal(cop, rcop) and np.array_equal(sp, rsp) and np.array_equal(cs, rcs)
    info = plan.info
    counts = np.diff(rcs)
    assert info.nz == nz and info.n_cells == rig.n_cells * nz
    assert info.n_column + info.n_generic == int((counts > 0).sum())
    assert info.n_empty == int((counts == 0).sum())
    plan.close()


@pytest.mark.parametrize("name", ["nuscenes", "nuscenes_tilted"])
def test_slab_forward_bf16_and_batch(torch_cuda, pkg, oracle_lib, name):
    """Four slabs, bf16 inputs, two frames in one call, against the oracle
    (reduced-precision bound of the forward: 2e-2 of the sum of |terms|)."""
    _say(f"[slab bf16 batch] {name}")
    torch = torch_cuda
    rig = dataclasses.replace(RIGS[name](), z_min=-8.0, z_cell=4.0)
    C, nz = 24, 4
    Pd, Fd, Ph, Fh = _inputs(torch, rig, C, seed=53, dtype="bf16", batch=2)
    sp = pkg.SlabPlan.from_rig(rig, nz)
    got = sp.forward(Pd, Fd).cpu().numpy().astype(np.float64)
    grid = oracle_lib.slab_grid(rig, nz)
    cop = oracle_lib.cell_map(rig, nz)
    _, ref, scale = oracle_lib.pool(grid, cop, Ph, Fh, want_f64=True, want_abs=True)
    ref = ref.reshape(got.shape)
    scale = scale.reshape(got.shape)
    assert (np.abs(got - ref) <= 2e-2 * scale + 1e-6).all()
    sp.close()


def test_slab_backward(torch_cuda, pkg, oracle_lib):
    """Gradients through a plan of three slabs against the oracle's, on the
    widened grid (|dP - ref| <= 1e-4 sqrt(C), |dF - ref| <= 1e-4 sqrt(k))."""
    _say("[slab backward]")
    torch = torch_cuda
    rig = dataclasses.replace(RIGS["nuscenes"](), z_min=-6.0, z_cell=4.0)
    C, nz = 16, 3
    Pd, Fd, Ph, Fh = _inputs(torch, rig, C, seed=57)
    G = np.random.default_rng(58).standard_normal((1, rig.ny, rig.nx, nz * C)).astype(np.float32)
    sp = pkg.SlabPlan.from_rig(rig, nz)
    gd, gf = sp.backward(torch.from_numpy(G).cuda(), Pd, Fd)
    grid = oracle_lib.slab_grid(rig, nz)
    cop = oracle_lib.cell_map(rig, nz)
    refP, refF = oracle_lib.backward(grid, cop, Ph, Fh, G.reshape(1, rig.ny, rig.nx * nz, C))
    errP = np.abs(gd.cpu().numpy().reshape(-1).astype(np.float64) - refP.reshape(-1))
    assert (errP <= 1e-4 * np.sqrt(C)).all(), errP.max()
    k = (cop >= 0).reshape(rig.n_cams, rig.n_depth, -1).sum(axis=1).reshape(-1)
    errF = np.abs(gf.cpu().numpy().reshape(rig.n_pixels, C).astype(np.float64) - refF.reshape(rig.n_pixels, C))
    assert (errF <= 1e-4 * np.sqrt(np.maximum(k, 1))[:, None]).all(), errF.max()
    sp.close()
