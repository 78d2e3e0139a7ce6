"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

- Plan: cell_of_point, sorted_point and cell_start must match bit for bit.
- fp32 forward: every element within 1e-4 * sqrt(points in its cell), and
  cells with no kept point exactly 0.
- bf16 / fp16 inputs: both sides read the same rounded values. The bound is
  2e-2 * sum |P * F| + 1e-6 per element, and the fp32 bound above must hold too.
"""
import dataclasses
import os
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


def _coarse_rig():
    """The nuScenes rig on a 3 m grid: cells with thousands of points, each
    fed by many combos (partial-sum slots added by the second kernel)."""
    return dataclasses.replace(wl.ring_rig(), nx=36, ny=36, cell_x=3.0, cell_y=3.0)


def _coarse_tilted_rig():
    """The tilted rig on a 3 m grid: generic cells with thousands of points,
    summed by a whole workgroup over many 64-run chunks."""
    return dataclasses.replace(wl.tilt_rig(wl.ring_rig()), nx=36, ny=36, cell_x=3.0, cell_y=3.0)


def _anisotropic_rig():
    base = wl.tilt_rig(wl.ring_rig(), 3.0, -4.0)
    intr = np.array([[35.0, 47.0, 21.5, 7.25], [41.0, 29.0, 24.0, 9.5]])
    return dataclasses.replace(base, n_cams=2, feat_h=16, feat_w=44, n_depth=40,
                               depth_min=0.75, depth_step=1.3, nx=150, ny=90,
                               x_min=-40.0, y_min=-20.0, cell_x=0.55, cell_y=0.45,
                               z_min=-1.0, z_cell=3.5, intrinsics=intr,
                               extrinsics=base.extrinsics[[1, 4]].copy())


def _odd_rig(tilt: bool):
    """Three cameras of the ring with odd sizes everywhere (13 rows, 27
    columns, 37 depth bins, a 151 x 149 grid): ragged row passes, column
    blocks and depth blocks; tilted, it also has generic cells."""
    base = wl.ring_rig()
    intr = base.intrinsics[[0, 2, 4]].copy()
    intr[:, 0] *= 27 / 88
    intr[:, 1] *= 13 / 32
    intr[:, 2] = 27 / 2
    intr[:, 3] = 13 / 2
    rig = dataclasses.replace(base, n_cams=3, feat_h=13, feat_w=27, n_depth=37, depth_min=1.0,
                              depth_step=1.5, nx=151, ny=149, x_min=-45.3, y_min=-44.7,
                              cell_x=0.6, cell_y=0.6, intrinsics=intr,
                              extrinsics=base.extrinsics[[0, 2, 4]].copy())
    return wl.tilt_rig(rig, 4.0, -3.0) if tilt else rig


def _empty_rig():
    return dataclasses.replace(wl.tiny_rig(), x_min=100.0)      # grid far from the camera


def _one_cell_rig():
    return dataclasses.replace(wl.tiny_rig(), nx=1, ny=1, x_min=0.0, y_min=-8.0,
                               cell_x=16.0, cell_y=16.0)


def _ring20_rig():
    """Twenty level cameras on the ring (more than the 16 whose calibration
    the plan build passes in kernel arguments, so it is copied to the device
    instead), 8x16 features, 24 depth bins, a 120 x 120 grid at 0.9 m."""
    H, W, N = 8, 16, 20
    intr = np.tile(np.array([[14.0, 14.0, W / 2.0, H / 2.0]]), (N, 1))
    return dataclasses.replace(wl.ring_rig(), n_cams=N, feat_h=H, feat_w=W, n_depth=24,
                               depth_min=1.0, depth_step=2.0, nx=120, ny=120, cell_x=0.9,
                               cell_y=0.9, intrinsics=intr,
                               extrinsics=wl._ring_extrinsics(N, 1.0, 1.5))


def _tall_rig():
    """The tiny camera with a feature map of 16,400 rows (more than the 2^14
    that the column table's row fields hold), 3 columns and 3 depth bins:
    every combo is geometrically clean (a level camera), but no combo can be
    column-served, so every cell takes the gathered path (16,400 or 32,800
    points each)."""
    H, W = 16400, 3
    return dataclasses.replace(wl.tiny_rig(), feat_h=H, feat_w=W, n_depth=3,
                               intrinsics=np.array([[1.5, H / 2.0, W / 2.0, H / 2.0]]))


RIGS = {
    "tiny": wl.tiny_rig, "tiny_identity": wl.identity_rig, "nuscenes": wl.ring_rig,
    "nuscenes_tilted": lambda: wl.tilt_rig(wl.ring_rig()), "highres": lambda: wl.ring_rig(2),
    # a calibration-sized tilt: combos split into row segments, one pass each
    "nuscenes_tilt1": lambda: wl.tilt_rig(wl.ring_rig(), 1.0, 0.5),
    "anisotropic": _anisotropic_rig, "coarse": _coarse_rig, "coarse_tilted": _coarse_tilted_rig,
    "empty": _empty_rig,
    "odd": lambda: _odd_rig(False), "odd_tilted": lambda: _odd_rig(True),
    "one_cell": _one_cell_rig, "tall": _tall_rig, "ring20": _ring20_rig,
}


@pytest.fixture(scope="module")
def oracle_plans(oracle_lib):
    cache = {}

    def get(name):
        if name not in cache:
            cache[name] = oracle_lib.plan(RIGS[name]())
        return cache[name]
    return get


@pytest.mark.parametrize("name", list(RIGS))
def test_plan_bit_exact(pkg, oracle_plans, name):
    _say(f"[plan] {name}")
    rig = RIGS[name]()
    plan = pkg.Plan.from_rig(rig)
    cop, sp, cs = plan.export()
    rcop, rsp, rcs = oracle_plans(name)
    assert np.array_equal(cop, rcop)
    assert np.array_equal(sp, rsp)
    assert np.array_equal(cs, rcs)
    counts = np.diff(rcs)
    assert plan.info.n_kept == rsp.size
    assert plan.info.n_nonempty == int((counts > 0).sum())
    assert plan.info.max_per_cell == int(counts.max(initial=0))
    assert plan.info.n_points == rig.n_points and plan.info.n_cells == rig.n_cells
    plan.close()


def _to_device(torch, arr, dtype):
    t = torch.from_numpy(np.ascontiguousarray(arr)).cuda()
    return t.to({"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[dtype])


def _check_fp32(got, ref, counts):
    """|got - ref| <= 1e-4 sqrt(count) per element; empty cells exactly 0."""
    B = got.shape[0]
    g = got.reshape(B, counts.size, -1)
    r = ref.reshape(B, counts.size, -1)
    bound = 1e-4 * np.sqrt(np.maximum(counts, 1))[None, :, None]
    err = np.abs(g.astype(np.float64) - r.astype(np.float64))
    worst = float((err / bound).max()) if err.size else 0.0
    assert (err <= bound).all(), f"max err/bound {worst:.3g}"
    assert (g[:, counts == 0] == 0).all()
    return worst


def _run(torch, pkg, plan, w):
    P = _to_device(torch, w.P, w.dtype)
    F = _to_device(torch, w.F, w.dtype)
    out = plan.forward(P, F)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("name,seed", [("tiny", 0), ("tiny_identity", 1), ("nuscenes", 0),
                                       ("nuscenes_tilted", 2)])
def test_forward_fp32(torch_cuda, pkg, oracle_lib, oracle_plans, name, seed):
    _say(f"[forward fp32] {name} seed={seed}")
    w = wl.make(name, seed=seed)
    cop, _, cs = oracle_plans(name)
    ref = oracle_lib.pool(w.rig, cop, w.P, w.F)
    plan = pkg.Plan.from_rig(w.rig)
    got = _run(torch_cuda, pkg, plan, w)
    worst = _check_fp32(got, ref, np.diff(cs))
    _say(f"  worst err/bound {worst:.3g}")


@pytest.mark.parametrize("name,rig_name", [("nuscenes_bf16", "nuscenes"), ("nuscenes_f16", "nuscenes"),
                                           ("nuscenes_bf16", "nuscenes_tilt1"),
                                           ("nuscenes_f16", "nuscenes_tilt1")])
def test_forward_reduced_precision(torch_cuda, pkg, oracle_lib, oracle_plans, name, rig_name):
    """bf16 / fp16 inputs, fp32 accumulation, on the level rig and on the
    slightly tilted one (row segments)."""
    _say(f"[forward {name} on {rig_name}]")
    w = wl.make(name, seed=0)
    if rig_name != "nuscenes":
        w = dataclasses.replace(w, rig=RIGS[rig_name]())
    cop, _, cs = oracle_plans(rig_name)
    ref, ref64, abs64 = oracle_lib.pool(w.rig, cop, w.P, w.F, want_f64=True, want_abs=True)
    plan = pkg.Plan.from_rig(w.rig)
    got = _run(torch_cuda, pkg, plan, w)
    err = np.abs(got.astype(np.float64) - ref64)
    assert (err <= 2e-2 * abs64 + 1e-6).all()
    _check_fp32(got, ref, np.diff(cs))
    rel = np.linalg.norm(got - ref64) / np.linalg.norm(ref64)
    _say(f"  global relative L2 error {rel:.3g}")


@pytest.mark.parametrize("rig_name", ["nuscenes", "nuscenes_tilt1"])
def test_forward_batched_matches_single_frames(torch_cuda, pkg, oracle_lib, oracle_plans, rig_name):
    _say(f"[forward batched] 8 frames on {rig_name}")
    torch = torch_cuda
    w = wl.make("nuscenes_b8", seed=0)
    if rig_name != "nuscenes":
        w = dataclasses.replace(w, rig=RIGS[rig_name]())
    cop, _, cs = oracle_plans(rig_name)
    plan = pkg.Plan.from_rig(w.rig)
    P = _to_device(torch, w.P, "f32")
    F = _to_device(torch, w.F, "f32")
    batched = plan.forward(P, F).cpu().numpy()
    for b in range(w.batch):
        single = plan.forward(P[b:b + 1].contiguous(), F[b:b + 1].contiguous()).cpu().numpy()
        assert np.array_equal(batched[b:b + 1], single)
    ref = oracle_lib.pool(w.rig, cop, w.P, w.F)
    _check_fp32(batched, ref, np.diff(cs))


def test_forward_highres(torch_cuda, pkg, oracle_lib, oracle_plans):
    _say("[forward highres] 6x236x64x176 C=128 -> 720x720")
    w = wl.make("highres", seed=0)
    cop, _, cs = oracle_plans("highres")
    ref = oracle_lib.pool(w.rig, cop, w.P, w.F)
    plan = pkg.Plan.from_rig(w.rig)
    got = _run(torch_cuda, pkg, plan, w)
    _check_fp32(got, ref, np.diff(cs))


@pytest.mark.parametrize("name", ["coarse", "coarse_tilted", "anisotropic", "empty", "one_cell",
                                  "odd", "odd_tilted", "tall", "ring20"])
def test_forward_edge_rigs(torch_cuda, pkg, oracle_lib, oracle_plans, name):
    _say(f"[forward edge] {name}")
    rig = RIGS[name]()
    P, F = wl.frames(rig, 16, 1, "normal", seed=5)
    w = wl.Workload(name, rig, 16, 1, "f32", P, F)
    cop, _, cs = oracle_plans(name)
    ref = oracle_lib.pool(rig, cop, P, F)
    plan = pkg.Plan.from_rig(rig)
    got = _run(torch_cuda, pkg, plan, w)
    _check_fp32(got, ref, np.diff(cs))
    if name == "coarse":
        assert plan.info.max_per_cell > 1536
        # cells fed by many combos: partial sums in borrowed empty rows, or
        # (when the grid has too few empty rows) the generic path
        assert plan.info.n_partials > 0 or plan.info.n_generic > 0
        assert plan.info.n_partials <= plan.info.n_empty
    if name == "coarse_tilted":
        assert plan.info.n_generic > 0 and plan.info.max_per_cell > 1536   # heavy generic cells
    if name == "empty":
        assert plan.info.n_kept == 0 and (got == 0).all()
    if name.startswith("odd"):
        assert plan.info.n_kept > 0 and plan.info.n_column > 0
        if name == "odd_tilted":
            assert plan.info.n_generic > 0
    if name == "ring20":
        assert plan.info.n_kept > 0 and plan.info.n_column > 0
    if name == "tall":
        counts = np.diff(cs)
        assert plan.info.n_column == 0 and plan.info.n_generic == int((counts > 0).sum())
        assert plan.info.max_per_cell == int(counts.max()) >= rig.feat_h


@pytest.mark.parametrize("rig_name", ["nuscenes", "nuscenes_tilted", "nuscenes_tilt1"])
@pytest.mark.parametrize("channels", [1, 3, 5, 12, 17, 33, 64, 72, 81, 128, 160, 192, 260])
def test_forward_channel_counts(torch_cuda, pkg, oracle_lib, oracle_plans, channels, rig_name):
    """Every lane-chunk count (1..5 channels per lane of a 16-lane group),
    ragged last chunks, rows split into channel slices (81, 160, 260), and
    4-element lanes (72 and 160; 260 has slices of 65, which are not
    4-aligned). The level rig runs mostly column items, the tilted one mostly
    generic cells."""
    _say(f"[forward channels] {rig_name} C={channels}")
    rig = RIGS[rig_name]()
    P, F = wl.frames(rig, channels, 1, "peaked", seed=channels)
    w = wl.Workload("c", rig, channels, 1, "f32", P, F)
    cop, _, cs = oracle_plans(rig_name)
    ref = oracle_lib.pool(rig, cop, P, F)
    plan = pkg.Plan.from_rig(rig)
    _check_fp32(_run(torch_cuda, pkg, plan, w), ref, np.diff(cs))


def test_count_test_on_gpu(torch_cuda, pkg, oracle_plans):
    """P = 1, F = 1, C = 1: each cell holds its point count exactly."""
    torch = torch_cuda
    rig = wl.ring_rig()
    _, _, cs = oracle_plans("nuscenes")
    plan = pkg.Plan.from_rig(rig)
    P = torch.ones((1, rig.n_cams, rig.n_depth, rig.feat_h, rig.feat_w), device="cuda")
    F = torch.ones((1, rig.n_cams, rig.feat_h, rig.feat_w, 1), device="cuda")
    out = plan.forward(P, F).cpu().numpy().reshape(-1)
    assert np.array_equal(out, np.diff(cs).astype(np.float32))


def test_inputs_aligned_to_one_element(torch_cuda, pkg, oracle_lib, oracle_plans):
    torch = torch_cuda
    w = wl.make("nuscenes", seed=3)
    cop, _, cs = oracle_plans("nuscenes")
    ref = oracle_lib.pool(w.rig, cop, w.P, w.F)
    plan = pkg.Plan.from_rig(w.rig)
    P = _to_device(torch, w.P, "f32")
    flat = torch.empty(w.F.size + 1, device="cuda")
    flat[1:] = torch.from_numpy(w.F.reshape(-1)).cuda()
    F = flat[1:].view(w.F.shape)                  # 4-byte aligned only
    out = plan.forward(P, F)
    torch.cuda.synchronize()
    _check_fp32(out.cpu().numpy(), ref, np.diff(cs))
    # the output 4-byte aligned only as well, and the features aligned again
    oflat = torch.full((out.numel() + 1,), float("nan"), device="cuda")
    out2 = oflat[1:].view(out.shape)
    plan.forward(P, _to_device(torch, w.F, "f32"), out=out2)
    torch.cuda.synchronize()
    _check_fp32(out2.cpu().numpy(), ref, np.diff(cs))


def test_deterministic(torch_cuda, pkg):
    torch = torch_cuda
    w = wl.make("nuscenes_tilted", seed=6)
    plan = pkg.Plan.from_rig(w.rig)
    P = _to_device(torch, w.P, "f32")
    F = _to_device(torch, w.F, "f32")
    a = plan.forward(P, F).cpu().numpy()
    b = plan.forward(P, F).cpu().numpy()
    assert np.array_equal(a, b)


@pytest.mark.parametrize("name", ["tiny", "nuscenes", "nuscenes_tilted", "nuscenes_tilt1", "coarse",
                                  "empty"])
def test_plan_import_round_trip(torch_cuda, pkg, name):
    """A plan rebuilt from its exported cell map (bevpool_plan_import) has
    the same association, the same partition and the same pooled map, bit
    for bit, as the plan built from the calibration."""
    torch = torch_cuda
    print(f"[import] {name}", flush=True)
    rig = RIGS[name]()
    a = pkg.Plan.from_rig(rig)
    cop, sp, cs = a.export()
    b = pkg.Plan.from_cells(cop, rig)
    cop2, sp2, cs2 = b.export()
    assert np.array_equal(cop, cop2) and np.array_equal(sp, sp2) and np.array_equal(cs, cs2)
    for f, _ in pkg._binding.bevpool_plan_info._fields_:
        assert getattr(a.info, f) == getattr(b.info, f), f
    P, F = wl.frames(rig, 16, 1, "peaked", seed=4)
    Pd, Fd = _to_device(torch, P, "f32"), _to_device(torch, F, "f32")
    assert torch.equal(a.forward(Pd, Fd), b.forward(Pd, Fd))
    a.close()
    b.close()


@pytest.mark.parametrize("rig_name", ["nuscenes", "nuscenes_tilt1"])
def test_one_plan_on_two_streams(torch_cuda, pkg, rig_name):
    """The plan is read-only during a forward: two streams pool different
    frames with it at once (each into its own map), several times over, and
    every map equals the one pooled alone."""
    torch = torch_cuda
    _say(f"[two streams] {rig_name}")
    w = wl.make("nuscenes", seed=12, batch=2)
    if rig_name != "nuscenes":
        w = dataclasses.replace(w, rig=RIGS[rig_name]())
    plan = pkg.Plan.from_rig(w.rig)
    P = _to_device(torch, w.P, "f32")
    F = _to_device(torch, w.F, "f32")
    ref = [plan.forward(P[b:b + 1].contiguous(), F[b:b + 1].contiguous()) for b in range(2)]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    ins = [(P[b:b + 1].contiguous(), F[b:b + 1].contiguous()) for b in range(2)]
    torch.cuda.synchronize()
    outs = [[], []]
    for _ in range(4):
        for b, s in enumerate(streams):
            with torch.cuda.stream(s):
                outs[b].append(plan.forward(*ins[b], stream=s))
    torch.cuda.synchronize()
    for b in range(2):
        for o in outs[b]:
            assert torch.equal(o, ref[b])
    plan.close()


def test_plan_reuse_and_shape_checks(torch_cuda, pkg):
    torch = torch_cuda
    rig = wl.tiny_rig()
    plan = pkg.Plan.from_rig(rig)
    P = torch.zeros((1, 1, 8, 4, 8), device="cuda")
    F = torch.zeros((1, 1, 4, 8, 8), device="cuda")
    with pytest.raises(pkg.BevpoolError):
        plan.forward(P[:, :, :7].contiguous(), F)
    with pytest.raises(pkg.BevpoolError):
        plan.forward(P, F.to(torch.float16))
    assert (plan.forward(P, F) == 0).all()


def test_plan_used_on_another_device_is_rejected(torch_cuda, pkg):
    """A plan's arrays live on the device it was built on: the forward and the
    backward refuse to run when the current device differs. One GPU cannot
    make another device current, so the test marks the plan as built on
    device 7 (the int after the handle's 32-bit magic), checks the refusal
    before any launch, and restores the field."""
    import ctypes
    torch = torch_cuda
    plan = pkg.Plan.from_rig(wl.tiny_rig())
    P = torch.zeros((1, 1, 8, 4, 8), device="cuda")
    F = torch.zeros((1, 1, 4, 8, 8), device="cuda")
    G = torch.zeros((1, 16, 16, 8), device="cuda")
    dev = ctypes.c_int.from_address(plan.handle + 4)
    assert dev.value == torch.cuda.current_device()
    dev.value = 7
    try:
        with pytest.raises(pkg.BevpoolError, match="device 7"):
            plan.forward(P, F)
        with pytest.raises(pkg.BevpoolError, match="device 7"):
            plan.backward(G, P, F)
    finally:
        dev.value = torch.cuda.current_device()
    assert (plan.forward(P, F) == 0).all()
    plan.close()


@pytest.mark.parametrize("name", ["nuscenes", "nuscenes_tilted", "nuscenes_tilt1", "coarse",
                                  "anisotropic", "tiny", "tall"])
def test_plan_partition_counts(pkg, oracle_plans, name):
    """Every cell is column-served, generic or empty; the level rig has no
    generic cell at all."""
    rig = RIGS[name]()
    plan = pkg.Plan.from_rig(rig)
    info = plan.info
    counts = np.diff(oracle_plans(name)[2])
    assert info.n_column + info.n_generic == int((counts > 0).sum())
    assert info.n_empty == int((counts == 0).sum())
    assert info.n_runs >= info.n_generic
    assert info.n_partials <= info.n_empty
    if name == "nuscenes_tilt1":
        # every combo's kept rows fall into at most four segments of one
        # cell each, so the column items serve every cell (whole combos
        # alone would leave most cells generic)
        assert info.n_generic == 0 and info.n_column == int((counts > 0).sum())
    if name == "nuscenes":
        # a level rig: every combo is clean, so the partial slots are the
        # combos of cells whose kept points come from two or more (n, d, w)
        # combos
        cop, sp, cs = oracle_plans(name)
        H, W, D = rig.feat_h, rig.feat_w, rig.n_depth
        p = sp[:cs[-1]].astype(np.int64)
        combo = (p // (H * W)) * W + p % W                  # (n * D + d) * W + w
        pairs = np.unique(cop[p].astype(np.int64) * (rig.n_cams * D * W) + combo)
        per_cell = np.bincount(pairs // (rig.n_cams * D * W), minlength=rig.n_cells)
        assert info.n_generic == 0
        assert info.n_partials == int(per_cell[per_cell > 1].sum())   # one slot per combo
        assert info.n_multi == int((per_cell > 1).sum())
    plan.close()


def test_forward_timed_matches_forward(torch_cuda, pkg):
    """bevpool_forward_timed gives the same bits as bevpool_forward and a
    positive kernel-boundary time."""
    torch = torch_cuda
    w = wl.make("nuscenes", seed=4)
    plan = pkg.Plan.from_rig(w.rig)
    P = _to_device(torch, w.P, "f32")
    F = _to_device(torch, w.F, "f32")
    a = plan.forward(P, F)
    ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    b = plan.forward(P, F, events=ev)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    assert ev[0].elapsed_time(ev[1]) > 0.0
    plan.close()
