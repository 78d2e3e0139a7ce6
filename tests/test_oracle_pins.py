"""Pins of the CPU oracle to things other than itself (CPU only).

Each test holds the oracle to a closed form, a library routine taking a
different computational route, or an invariant of the definition in the
paper (BEVFusion, Sec. III-B). None of them re-types the oracle's formulas.
"""
import dataclasses
import os
import subprocess
import sys

import numpy as np
import pytest

import workloads as wl

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _read_golden(name):
    rows = {}
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, _, val = line.partition(":") if ":" in line else line.partition(" ")
            rows[key.strip()] = val.split()
    return rows


def _decode(rig, p):
    """(n, d, h, w) of point ids p = ((n*D + d)*H + h)*W + w."""
    w = p % rig.feat_w
    h = (p // rig.feat_w) % rig.feat_h
    d = (p // (rig.feat_w * rig.feat_h)) % rig.n_depth
    n = p // (rig.feat_w * rig.feat_h * rig.n_depth)
    return n, d, h, w


# ------------------------------------------------------------------ plan pins

def test_paper_typical_workload_point_count():
    """The nuScenes-shaped rig has the paper's N, H, W, D and about 2 M points
    (Sec. III-B footnote)."""
    g = _read_golden("paper_typical_workload.txt")
    rig = wl.ring_rig()
    assert rig.n_cams == int(g["n_cams"][0])
    assert (rig.feat_h, rig.feat_w) == (int(g["feat_h"][0]), int(g["feat_w"][0]))
    D = (float(g["depth_max"][0]) - float(g["depth_min"][0])) / float(g["depth_step"][0])
    assert rig.n_depth == int(g["n_depth"][0]) == int(D)
    assert rig.depth_min == float(g["depth_min"][0])
    assert rig.depth_step == float(g["depth_step"][0])
    assert rig.n_points == 1_993_728
    assert abs(rig.n_points - int(g["approx_points"][0])) / 2e6 < 0.01


def test_tiny_rig_closed_form(oracle_lib):
    """Tiny rig: ego x = d, y = d(7-2w)/8, so ix = d + 8 and
    iy = floor(8 + d(7-2w)/8); d = 8 sits on the open upper edge."""
    rig = wl.tiny_rig()
    cop = oracle_lib.cell_map(rig)
    g = _read_golden("tiny_rig_closed_form.txt")
    p = np.arange(rig.n_points)
    _, k, h, w = _decode(rig, p)
    depth = k + 1
    for dd in range(1, 8):
        expect_iy = np.array([int(v) for v in g[f"iy d={dd}"]])
        sel = depth == dd
        cells = cop[sel]
        assert (cells >= 0).all()
        assert (cells % 16 == dd + 8).all()
        assert (cells // 16 == expect_iy[w[sel]]).all()
    assert (cop[depth == 8] == -1).all()
    counts = np.bincount(cop[cop >= 0], minlength=rig.n_cells)
    assert (cop >= 0).sum() == int(g["kept"][0])
    assert (counts > 0).sum() == int(g["nonempty"][0])
    assert counts.max() == int(g["max_per_cell"][0])


def test_identity_rig_closed_form(oracle_lib):
    """Identity extrinsics: x = d(2w-7)/8, y = d(2h-3)/8, z = d, all exact
    dyadics, so ix = floor((64 + d(2w-7))/8) in integer arithmetic."""
    rig = wl.identity_rig()
    cop = oracle_lib.cell_map(rig)
    n, k, h, w = _decode(rig, np.arange(rig.n_points))
    d = k + 1
    ix = (64 + d * (2 * w - 7)) // 8
    iy = (64 + d * (2 * h - 3)) // 8
    assert (cop == iy * 16 + ix).all()
    counts = np.bincount(cop, minlength=rig.n_cells)
    assert (counts > 0).sum() == 86 and counts.max() == 18


def _linalg_cells(rig, nz=1):
    """Cells through a different route: 3x3 intrinsic matrix inverted by
    numpy.linalg, 4x4 homogeneous extrinsic, matrix products. Returns the
    cell ids and a mask of points whose quantised coordinates sit within
    1e-9 (relative) of a cell edge, where rounding may legitimately differ.
    With nz slabs the cell id is (iy * nx + ix) * nz + iz."""
    N, D, H, W = rig.n_cams, rig.n_depth, rig.feat_h, rig.feat_w
    cells = np.empty(rig.n_points, dtype=np.int64)
    near = np.zeros(rig.n_points, dtype=bool)
    hh, ww = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    pix = np.stack([ww.ravel() + rig.pixel_offset, hh.ravel() + rig.pixel_offset,
                    np.ones(H * W)])                                   # 3 x HW
    depths = rig.depth_min + np.arange(D) * rig.depth_step
    for n in range(N):
        fx, fy, cx, cy = rig.intrinsics[n]
        K = np.array([[fx, 0.0, cx], [0.0, fy, cy], [0.0, 0.0, 1.0]])
        T = np.eye(4)
        T[:3, :] = rig.extrinsics[n].reshape(3, 4)
        rays = np.linalg.inv(K) @ pix                                  # 3 x HW
        pts = rays[None, :, :] * depths[:, None, None]                 # D x 3 x HW
        hom = np.concatenate([pts, np.ones((D, 1, H * W))], axis=1)    # D x 4 x HW
        ego = np.einsum("ij,djk->dik", T, hom)[:, :3, :]
        q = np.stack([(ego[:, 0] - rig.x_min) / rig.cell_x,
                      (ego[:, 1] - rig.y_min) / rig.cell_y,
                      (ego[:, 2] - rig.z_min) / rig.z_cell])
        fl = np.floor(q)
        frac = np.minimum(q - fl, fl + 1 - q)
        close = (frac < 1e-9 * np.maximum(1.0, np.abs(q))).any(axis=0)
        keep = ((fl[0] >= 0) & (fl[0] < rig.nx) & (fl[1] >= 0) & (fl[1] < rig.ny) & (fl[2] >= 0)
                & (fl[2] < nz))
        c = np.where(keep, (fl[1] * rig.nx + fl[0]) * nz + fl[2], -1).astype(np.int64)
        sl = slice(n * D * H * W, (n + 1) * D * H * W)
        cells[sl] = c.reshape(-1)
        near[sl] = close.reshape(-1)
    return cells, near


def _anisotropic_rig():
    """Two cameras with fx != fy, a non-square grid and unequal cell sides,
    so a swapped axis or index shows."""
    base = wl.tilt_rig(wl.ring_rig(), 3.0, -4.0)
    intr = np.array([[35.0, 47.0, 21.5, 7.25], [41.0, 29.0, 24.0, 9.5]])
    return dataclasses.replace(base, n_cams=2, feat_h=16, feat_w=44, n_depth=40,
                               depth_min=0.75, depth_step=1.3, nx=150, ny=90,
                               x_min=-40.0, y_min=-20.0, cell_x=0.55, cell_y=0.45,
                               z_min=-1.0, z_cell=3.5, intrinsics=intr,
                               extrinsics=base.extrinsics[[1, 4]].copy())


@pytest.mark.parametrize("rigname", ["nuscenes", "nuscenes_tilted", "anisotropic"])
def test_cells_match_homogeneous_matrix_route(oracle_lib, rigname):
    rig = _anisotropic_rig() if rigname == "anisotropic" else wl.WORKLOADS[rigname][0]()
    cop = oracle_lib.cell_map(rig)
    ref, near = _linalg_cells(rig)
    # the level ring rig puts every third depth bin of the cameras at yaw 0
    # and 180 degrees exactly on a cell edge; those points are decided by
    # rounding alone and are left out of this comparison
    assert near.mean() < 0.15
    assert (cop[~near] == ref[~near]).all()
    assert 0.1 < (cop >= 0).mean() < 1.0


def test_z_slab_filter(oracle_lib):
    """Identity rig has z = d; with the slab [2, 6) only d = 2..5 survive."""
    rig = dataclasses.replace(wl.identity_rig(), z_min=2.0, z_cell=4.0)
    cop = oracle_lib.cell_map(rig)
    _, k, _, _ = _decode(rig, np.arange(rig.n_points))
    assert ((cop >= 0) == ((k + 1 >= 2) & (k + 1 < 6))).all()


def test_half_open_edges_and_floor(oracle_lib):
    """At d = 8 the identity rig puts x at the odd integers -7..7.
    With x_min = -7 and 14 cells, x = -7 is kept (closed lower edge) and
    x = 7 dropped (open upper edge). With x_min = -6.5, x = -7 lies half a
    cell below the grid and must be dropped (floor, not truncation)."""
    base = dataclasses.replace(wl.identity_rig(), n_depth=1, depth_min=8.0)
    _, _, h, w = _decode(base, np.arange(base.n_points))
    r1 = dataclasses.replace(base, x_min=-7.0, nx=14)
    c1 = oracle_lib.cell_map(r1)
    ix = 2 * w - 7 + 7                       # x - x_min with x = 2w - 7
    assert ((c1 >= 0) == (ix < 14)).all()
    assert (c1[ix < 14] % 14 == ix[ix < 14]).all()
    r2 = dataclasses.replace(base, x_min=-6.5, nx=14)
    c2 = oracle_lib.cell_map(r2)
    assert (c2[w == 0] == -1).all()            # x = -7: floor(-0.5) = -1
    assert (c2[w == 1] % 14 == 1).all()        # x = -5: floor(1.5) = 1


def test_sort_matches_lexsort(oracle_lib):
    rig = wl.tilt_rig(wl.ring_rig())
    cop, sp, cs = oracle_lib.plan(rig)
    ids = np.arange(rig.n_points)
    kept = cop >= 0
    order = np.lexsort((ids[kept], cop[kept]))
    assert (sp == ids[kept][order]).all()
    assert (cs == np.searchsorted(np.sort(cop[kept]), np.arange(rig.n_cells + 1))).all()


# ------------------------------------------------------------------ forward pins

def test_count_test(oracle_lib):
    """P = 1, F = 1, C = 1: every cell holds its point count, exactly."""
    rig = wl.ring_rig()
    cop, _, cs = oracle_lib.plan(rig)
    P = np.ones((1, rig.n_points), dtype=np.float32)
    F = np.ones((1, rig.n_pixels, 1), dtype=np.float32)
    out = oracle_lib.pool(rig, cop, P, F)
    assert (out.reshape(-1) == np.diff(cs)).all()
    assert (out.reshape(-1) == np.bincount(cop[cop >= 0], minlength=rig.n_cells)).all()


def _pixel_of(rig, p):
    n, _, h, w = _decode(rig, p)
    return (n * rig.feat_h + h) * rig.feat_w + w


@pytest.mark.parametrize("name", ["tiny", "tiny_identity"])
def test_dense_matrix_route(oracle_lib, name):
    """out = S @ (P * F[pixel]) with S the 0/1 cell-membership matrix."""
    w = wl.make(name, seed=3)
    rig = w.rig
    cop = oracle_lib.cell_map(rig)
    _, o64 = oracle_lib.pool(rig, cop, w.P, w.F, want_f64=True)
    p = np.arange(rig.n_points)
    S = np.zeros((rig.n_cells, rig.n_points))
    S[cop[cop >= 0], p[cop >= 0]] = 1.0
    terms = w.P[0].reshape(-1)[:, None].astype(np.float64) * \
        w.F[0].reshape(rig.n_pixels, -1)[_pixel_of(rig, p)].astype(np.float64)
    ref = S @ terms
    scale = S @ np.abs(terms) + 1e-300
    assert (np.abs(o64[0].reshape(rig.n_cells, -1) - ref) <= 1e-13 * scale).all()


@pytest.mark.parametrize("name", ["nuscenes_tilted"])
def test_sparse_matrix_route(oracle_lib, name):
    """The same product at full nuScenes size, through scipy.sparse."""
    import scipy.sparse as sps
    w = wl.make(name, seed=1)
    rig = w.rig
    cop = oracle_lib.cell_map(rig)
    _, o64 = oracle_lib.pool(rig, cop, w.P, w.F, want_f64=True)
    p = np.arange(rig.n_points)[cop >= 0]
    S = sps.csr_matrix((w.P[0].reshape(-1)[p].astype(np.float64), (cop[cop >= 0], _pixel_of(rig, p))),
                       shape=(rig.n_cells, rig.n_pixels))
    A = sps.csr_matrix((np.abs(w.P[0].reshape(-1)[p]).astype(np.float64), (cop[cop >= 0], _pixel_of(rig, p))),
                       shape=(rig.n_cells, rig.n_pixels))
    Fm = w.F[0].reshape(rig.n_pixels, -1).astype(np.float64)
    ref = S @ Fm
    scale = A @ np.abs(Fm) + 1e-300
    assert (np.abs(o64[0].reshape(rig.n_cells, -1) - ref) <= 1e-12 * scale).all()


def test_identity_onehot_exact(oracle_lib):
    """One-hot depth, identity extrinsics: each cell holds exactly the sum of
    the features of the pixels whose chosen bin lands there. Features are
    multiples of 2^-10, so every sum is exact in any order."""
    rig = wl.identity_rig()
    rng = np.random.default_rng(7)
    N, D, H, W, C = 1, rig.n_depth, rig.feat_h, rig.feat_w, 5
    kbin = rng.integers(0, D, size=(H, W))
    P = (np.arange(D)[:, None, None] == kbin[None]).astype(np.float32)[None, None]
    F = (np.round(rng.standard_normal((1, N, H, W, C)) * 1024) / 1024).astype(np.float32)
    cop = oracle_lib.cell_map(rig)
    out = oracle_lib.pool(rig, cop, P, F)
    expect = np.zeros((rig.n_cells, C))
    for h in range(H):
        for w_ in range(W):
            d = kbin[h, w_] + 1
            ix = (64 + d * (2 * w_ - 7)) // 8
            iy = (64 + d * (2 * h - 3)) // 8
            expect[iy * 16 + ix] += F[0, 0, h, w_].astype(np.float64)
    assert (out.reshape(rig.n_cells, C) == expect.astype(np.float32)).all()


def test_mass_conservation(oracle_lib):
    """All points kept and P a distribution over depth: the BEV total of each
    channel equals the image total of that channel."""
    w = wl.make("tiny_identity", seed=11)
    cop = oracle_lib.cell_map(w.rig)
    assert (cop >= 0).all()
    _, o64 = oracle_lib.pool(w.rig, cop, w.P, w.F, want_f64=True)
    psum = w.P[0].astype(np.float64).sum(axis=1)          # [N][H][W], ~1
    expect = (psum[..., None] * w.F[0].astype(np.float64)).sum(axis=(0, 1, 2))
    assert np.allclose(o64.sum(axis=(0, 1, 2)), expect, rtol=0, atol=1e-12 * np.abs(w.F).sum())
    assert np.allclose(psum, 1.0, atol=1e-6)


def test_camera_permutation_invariance(oracle_lib):
    """Relabelling cameras (calibration and data together) changes only the
    summation order."""
    w = wl.make("nuscenes", seed=2)
    rig = w.rig
    perm = np.array([3, 0, 5, 1, 4, 2])
    rig2 = dataclasses.replace(rig, intrinsics=rig.intrinsics[perm], extrinsics=rig.extrinsics[perm])
    _, a = oracle_lib.pool(rig, oracle_lib.cell_map(rig), w.P, w.F, want_f64=True)
    _, b = oracle_lib.pool(rig2, oracle_lib.cell_map(rig2), w.P[:, perm], w.F[:, perm], want_f64=True)
    assert np.allclose(a, b, rtol=0, atol=1e-12)


def test_channel_permutation_and_linearity(oracle_lib):
    w = wl.make("nuscenes_tilted", seed=4, channels=16)
    rig = w.rig
    cop = oracle_lib.cell_map(rig)
    _, base = oracle_lib.pool(rig, cop, w.P, w.F, want_f64=True)
    perm = np.random.default_rng(0).permutation(16)
    _, permuted = oracle_lib.pool(rig, cop, w.P, w.F[..., perm], want_f64=True)
    assert (permuted == base[..., perm]).all()
    _, doubled = oracle_lib.pool(rig, cop, w.P * 2, w.F, want_f64=True)
    assert (doubled == 2 * base).all()                      # power-of-two scale is exact
    F2 = np.random.default_rng(5).standard_normal(w.F.shape).astype(np.float32)
    _, o2 = oracle_lib.pool(rig, cop, w.P, F2, want_f64=True)
    _, o12 = oracle_lib.pool(rig, cop, w.P, w.F + F2, want_f64=True)
    _, scale = oracle_lib.pool(rig, cop, np.abs(w.P), np.abs(w.F) + np.abs(F2), want_f64=True)
    # F + F2 is rounded to float32 first: allow that rounding per term
    assert (np.abs(o12 - (base + o2)) <= 2 ** -23 * scale + 1e-300).all()


def test_thread_count_does_not_change_result(oracle_lib, tmp_path):
    """Channels are split across threads; each element's order is fixed."""
    code = (
        "import sys, numpy as np; sys.path.insert(0, %r)\n"
        "import oracle, workloads as wl\n"
        "w = wl.make('nuscenes_tilted', seed=9, channels=24)\n"
        "out = oracle.pool(w.rig, oracle.cell_map(w.rig), w.P, w.F)\n"
        "np.save(sys.argv[1], out)\n" % os.path.dirname(GOLDEN.rstrip('/')).rsplit('/', 1)[0])
    outs = []
    for threads in ("1", "3"):
        path = str(tmp_path / f"o{threads}.npy")
        env = dict(os.environ, OMP_NUM_THREADS=threads)
        subprocess.run([sys.executable, "-c", code, path], check=True, env=env)
        outs.append(np.load(path))
    assert (outs[0] == outs[1]).all()


# ---------------------------------------------------------------- gradients
#
# The pooling is bilinear in (P, F), so its gradients are pinned by the
# forward oracle itself (already pinned above) through identities that hold
# for any G, and by a Jacobian assembled from forward calls.

def _grad_inputs(name, seed, channels=None):
    w = wl.make(name, seed=seed, channels=channels) if channels else wl.make(name, seed=seed)
    rng = np.random.default_rng(seed + 100)
    G = rng.standard_normal((w.batch, w.rig.ny, w.rig.nx, w.channels)).astype(np.float32)
    return w, G


@pytest.mark.parametrize("name", ["tiny", "nuscenes_tilted", "nuscenes"])
def test_backward_adjoint_identities(oracle_lib, name):
    """<G, pool(P, F)> = <P, dP> = <F, dF>, each side in double."""
    w, G = _grad_inputs(name, seed=4)
    cop = oracle_lib.cell_map(w.rig)
    _, o64 = oracle_lib.pool(w.rig, cop, w.P, w.F, want_f64=True)
    dP, dF = oracle_lib.backward(w.rig, cop, w.P, w.F, G)
    lhs = float((G.astype(np.float64) * o64).sum())
    via_p = float((w.P.astype(np.float64) * dP).sum())
    via_f = float((w.F.astype(np.float64) * dF).sum())
    scale = float((np.abs(G).astype(np.float64) *
                   oracle_lib.pool(w.rig, cop, np.abs(w.P), np.abs(w.F), want_f64=True)[1]).sum())
    assert abs(lhs - via_p) <= 1e-12 * scale
    assert abs(lhs - via_f) <= 1e-12 * scale


@pytest.mark.parametrize("name", ["tiny", "tiny_identity"])
def test_backward_matches_forward_jacobian(oracle_lib, name):
    """Column p of d out / d P is pool with P = e_p; row-wise the same for F.
    The Jacobians are assembled from forward calls and contracted with G."""
    w, G = _grad_inputs(name, seed=5)
    rig = w.rig
    cop = oracle_lib.cell_map(rig)
    C = w.channels
    dP, dF = oracle_lib.backward(rig, cop, w.P, w.F, G)
    g64 = G[0].astype(np.float64).reshape(-1)
    for p in range(rig.n_points):
        e = np.zeros_like(w.P)
        e.reshape(-1)[p] = 1.0
        col = oracle_lib.pool(rig, cop, e, w.F, want_f64=True)[1].reshape(-1)
        assert abs(float(col @ g64) - dP.reshape(-1)[p]) <= 1e-12 * (np.abs(col) @ np.abs(g64) + 1e-300)
    for i in range(rig.n_pixels * C):
        e = np.zeros_like(w.F)
        e.reshape(-1)[i] = 1.0
        col = oracle_lib.pool(rig, cop, w.P, e, want_f64=True)[1].reshape(-1)
        assert abs(float(col @ g64) - dF.reshape(-1)[i]) <= 1e-12 * (np.abs(col) @ np.abs(g64) + 1e-300)


def test_backward_all_ones(oracle_lib):
    """G = 1 and F = 1: dP is C for every kept point and 0 for every dropped
    one; G = 1 and P = 1: dF[pixel][c] counts the pixel's kept depth bins."""
    rig = wl.ring_rig()
    cop = oracle_lib.cell_map(rig)
    C = 3
    ones_p = np.ones((1, rig.n_points), dtype=np.float32)
    ones_f = np.ones((1, rig.n_pixels, C), dtype=np.float32)
    ones_g = np.ones((1, rig.n_cells, C), dtype=np.float32)
    dP, dF = oracle_lib.backward(rig, cop, ones_p, ones_f, ones_g)
    assert (dP.reshape(-1) == np.where(cop >= 0, C, 0)).all()
    kept = (cop.reshape(rig.n_cams, rig.n_depth, rig.feat_h * rig.feat_w) >= 0).sum(axis=1)
    assert (dF.reshape(rig.n_pixels, C) == kept.reshape(-1)[:, None]).all()


# ------------------------------------------------------------------ mean / max pins

def _terms(w, cop):
    """(kept cells, exact double P * F of every kept point)."""
    rig = w.rig
    kept = cop >= 0
    p = np.arange(rig.n_points)[kept]
    terms = w.P[0].reshape(-1)[kept, None].astype(np.float64) * \
        w.F[0].reshape(rig.n_pixels, -1)[_pixel_of(rig, p)].astype(np.float64)
    return cop[kept], terms


@pytest.mark.parametrize("name,channels", [("tiny", None), ("tiny_identity", None),
                                           ("nuscenes_tilted", 6)])
def test_mean_max_numpy_ufunc_route(oracle_lib, name, channels):
    """Mean through numpy's add.at and bincount, max through maximum.at, over
    the cell map: library routines, no loop of ours. The max is exact (the
    same exact products), the mean agrees to double rounding."""
    w = wl.make(name, seed=5, channels=channels)
    rig = w.rig
    cop = oracle_lib.cell_map(rig)
    cells, terms = _terms(w, cop)
    C = terms.shape[1]
    cnt = np.bincount(cells, minlength=rig.n_cells)
    s = np.zeros((rig.n_cells, C))
    np.add.at(s, cells, terms)
    a = np.zeros((rig.n_cells, C))
    np.add.at(a, cells, np.abs(terms))
    m = np.full((rig.n_cells, C), -np.inf)
    np.maximum.at(m, cells, terms)
    has = cnt[:, None] > 0
    mean_ref = np.where(has, s / np.maximum(cnt, 1)[:, None], 0.0)
    max_ref = np.where(has, m, 0.0)
    mean = oracle_lib.pool_reduce(rig, cop, w.P, w.F, "mean")[0].reshape(rig.n_cells, C)
    mx = oracle_lib.pool_reduce(rig, cop, w.P, w.F, "max")[0].reshape(rig.n_cells, C)
    assert (mx == max_ref).all()
    scale = a / np.maximum(cnt, 1)[:, None] + 1e-300
    assert (np.abs(mean - mean_ref) <= 1e-13 * scale).all()
    assert (mean[~has[:, 0]] == 0).all() and (mx[~has[:, 0]] == 0).all()


def test_mean_max_tiny_golden():
    """Tiny rig, C = 1, F = 1 and P = (point id + 1) / 1024 (exact dyadics):
    each cell's max is its largest point id and its mean the mean id, both
    computed here from the hand-derived cell map in the golden file (a cell
    (ix, iy) holds the points with depth d = ix - 8 and any row h whose
    column w has iy in the table)."""
    import oracle
    rig = wl.tiny_rig()
    g = _read_golden("tiny_rig_closed_form.txt")
    H, W = rig.feat_h, rig.feat_w
    members = {}
    for dd in range(1, 8):
        iys = [int(v) for v in g[f"iy d={dd}"]]
        for wcol in range(W):
            cell = iys[wcol] * 16 + (dd + 8)
            for h in range(H):
                members.setdefault(cell, []).append(((dd - 1) * H + h) * W + wcol)
    exp_max = np.zeros(rig.n_cells)
    exp_mean = np.zeros(rig.n_cells)
    for cell, ids in members.items():
        exp_max[cell] = (max(ids) + 1) / 1024.0
        exp_mean[cell] = (sum(ids) + len(ids)) / len(ids) / 1024.0
    P = ((np.arange(rig.n_points) + 1) / 1024.0).astype(np.float32)[None]
    F = np.ones((1, rig.n_pixels, 1), dtype=np.float32)
    cop = oracle.cell_map(rig)
    mx = oracle.pool_reduce(rig, cop, P, F, "max").reshape(-1)
    mean = oracle.pool_reduce(rig, cop, P, F, "mean").reshape(-1)
    assert (mx == exp_max).all()
    assert np.allclose(mean, exp_mean, rtol=1e-15, atol=0)
    assert len(members) == int(g["nonempty"][0])


def test_min_mean_max_order(oracle_lib):
    """Per non-empty cell and channel: min <= mean <= max, with the min taken
    as -max of P * (-F)."""
    w = wl.make("nuscenes_tilted", seed=6, channels=4)
    cop = oracle_lib.cell_map(w.rig)
    mx = oracle_lib.pool_reduce(w.rig, cop, w.P, w.F, "max")
    mn = -oracle_lib.pool_reduce(w.rig, cop, w.P, -w.F, "max")
    mean = oracle_lib.pool_reduce(w.rig, cop, w.P, w.F, "mean")
    has = np.bincount(cop[cop >= 0], minlength=w.rig.n_cells).reshape(1, w.rig.ny, w.rig.nx, 1) > 0
    tol = 1e-12 * (np.abs(mx) + np.abs(mn))
    assert ((mn <= mean + tol) | ~has).all() and ((mean <= mx + tol) | ~has).all()
    assert (mn[has[..., 0]] < mx[has[..., 0]]).mean() > 0.5


# ------------------------------------------------------------------ z slab pins

def test_slabs_identity_rig_closed_form():
    """Identity rig (z = d exactly): four 2 m slabs from z = 0. Each kept
    point keeps the (x, y) cell of the single 8 m slab [0, 8), its slab is
    floor(d / 2), exactly the points of that 8 m slab are kept, and the
    slabs' sums add up to the sum over the 8 m slab."""
    import oracle
    w = wl.make("tiny_identity", seed=7)
    base = dataclasses.replace(w.rig, z_min=0.0, z_cell=2.0)
    union = dataclasses.replace(w.rig, z_min=0.0, z_cell=8.0)
    cu = oracle.cell_map(union)
    c4 = oracle.cell_map(base, 4)
    _, k, _, _ = _decode(base, np.arange(base.n_points))
    assert ((c4 >= 0) == (cu >= 0)).all() and ((cu >= 0) == (k + 1 < 8)).all()
    kept = c4 >= 0
    assert (c4[kept] // 4 == cu[kept]).all()
    assert (c4[kept] % 4 == (k[kept] + 1) // 2).all()
    cat = oracle.pool_slabs(base, 4, w.P, w.F)
    C = w.channels
    total = sum(cat[..., iz * C:(iz + 1) * C] for iz in range(4))
    _, ref = oracle.pool(union, cu, w.P, w.F, want_f64=True)
    _, a64 = oracle.pool(union, cu, np.abs(w.P), np.abs(w.F), want_f64=True)
    assert (np.abs(total - ref) <= 1e-13 * (a64 + 1e-300)).all()


def test_slabs_ring_rig_union():
    """nuScenes-shaped rig, four 4 m slabs from z = -8 m against the 16 m slab
    [-8, 8): the slab index divides z by 4 m, the union by 16 m (a power-of-
    two scaling), so the kept points agree exactly, and each keeps its cell."""
    import oracle
    rig = dataclasses.replace(wl.ring_rig(), z_min=-8.0, z_cell=4.0)
    cu = oracle.cell_map(dataclasses.replace(rig, z_cell=16.0))
    c4 = oracle.cell_map(rig, 4)
    assert ((c4 >= 0) == (cu >= 0)).all()
    assert (c4[c4 >= 0] // 4 == cu[cu >= 0]).all()
    assert len(np.unique(c4[c4 >= 0] % 4)) == 4
    assert 0.2 < (cu >= 0).mean() < 1.0


@pytest.mark.parametrize("rigname,nz", [("nuscenes", 4), ("nuscenes_tilted", 3), ("anisotropic", 5)])
def test_slab_cells_match_homogeneous_matrix_route(oracle_lib, rigname, nz):
    """The slab index and cell id through the numpy matrix route."""
    rig = _anisotropic_rig() if rigname == "anisotropic" else wl.WORKLOADS[rigname][0]()
    rig = dataclasses.replace(rig, z_min=rig.z_min, z_cell=rig.z_cell / nz)
    cop = oracle_lib.cell_map(rig, nz)
    ref, near = _linalg_cells(rig, nz)
    assert near.mean() < 0.15
    assert (cop[~near] == ref[~near]).all()
    kept = cop >= 0
    assert len(np.unique(cop[kept] % nz)) == nz


def test_one_slab_is_pool(oracle_lib):
    w = wl.make("tiny", seed=8)
    cop = oracle_lib.cell_map(w.rig)
    _, ref = oracle_lib.pool(w.rig, cop, w.P, w.F, want_f64=True)
    assert (oracle_lib.pool_slabs(w.rig, 1, w.P, w.F) == ref).all()
    ref_max = oracle_lib.pool_reduce(w.rig, cop, w.P, w.F, "max")
    assert (oracle_lib.pool_slabs(w.rig, 1, w.P, w.F, "max") == ref_max).all()
