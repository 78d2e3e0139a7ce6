"""CPU oracle for BEV pooling (BEVFusion, arXiv 2205.13542, Sec. III-B).

TEST INFRASTRUCTURE ONLY: the tests, the smoke entry point and the benchmark's
CPU-baseline leg may use it; the product path never does. It shares no code
with the GPU library (``paper_2205_13542_amd``) and imports nothing from it.

The arithmetic lives in ``bevpool_oracle.c`` (plain C, double precision,
built without FMA contraction or fast-math). This module builds it with gcc,
loads it with ctypes and marshals numpy arrays.

Functions and the passages they follow:

- ``cell_map``: grid index of every frustum point, -1 when dropped
  (Sec. III-B: lifting pixels to D points along the camera ray, quantising
  x and y at step r, one z slab; "Precomputation": the 3-D coordinate and
  grid index of each point).
- ``sort_by_cell``: points ordered by grid index, ties by point id, and the
  interval table ("Precomputation": sort by grid index and record ranks;
  "Interval Reduction": a cell's points are then consecutive).
- ``pool``: per-cell sums of P * F ("Interval Reduction": sum is one of the
  symmetric aggregations; "Takeaways": exact, no approximation).
- ``pool_reduce``: per-cell mean or max of P * F ("Interval Reduction": mean
  and max are the other symmetric aggregations it names); 0 for empty cells.
- ``pool_slabs``: several z slabs, each pooled on its own, concatenated
  along channels (Sec. III-B: flattening along z).
- ``backward``: the gradients of ``pool`` with respect to P and F for a given
  gradient of the BEV map (the pooling is one differentiable layer of a
  model trained end to end): dP[p] = F[pixel(p)] . G[cell(p)] and
  dF[pixel] = sum over its kept points of P[p] G[cell(p)].

Pins, i.e. what the tests hold this oracle to (none of them re-types its
formulas): closed-form cell maps of two dyadic rigs, a homogeneous-matrix
projection through numpy.linalg, numpy's lexsort, a dense 0/1 matrix
product, the count test, mass conservation, and permutation, linearity and
boundary cases; for the gradients, the adjoint identities
<G, pool(P, F)> = <P, dP> = <F, dF> against ``pool``, a dense Jacobian of
``pool`` built column by column on the tiny rig, and all-ones cases with
integer answers; for mean and max, numpy's ``add.at``/``bincount`` and
``maximum.at`` over the cell map, the golden cell maps of the tiny rig
(point-id probabilities give each cell's largest point id), and ordering
invariants; for slabs, the union of dyadic slabs against one slab of the
union's height. Values at the nuScenes-shaped sizes are pinned only by these
properties: the paper prints no pooled value (parity unpinned by the paper,
pinned by the invariants).
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "bevpool_oracle.c")
LIB_PATH = os.path.join(_HERE, "liboracle.so")

_lib = None


class _Geom(ctypes.Structure):
    _fields_ = [
        ("n_cams", ctypes.c_int32), ("feat_h", ctypes.c_int32),
        ("feat_w", ctypes.c_int32), ("n_depth", ctypes.c_int32),
        ("depth_min", ctypes.c_double), ("depth_step", ctypes.c_double),
        ("pixel_offset", ctypes.c_double),
        ("nx", ctypes.c_int32), ("ny", ctypes.c_int32),
        ("x_min", ctypes.c_double), ("y_min", ctypes.c_double),
        ("cell_x", ctypes.c_double), ("cell_y", ctypes.c_double),
        ("z_min", ctypes.c_double), ("z_cell", ctypes.c_double),
    ]


def build() -> str:
    """Compile the oracle with gcc (always, so a stale build never survives)."""
    tmp = LIB_PATH + ".tmp"
    cmd = ["gcc", "-O3", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
           "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        build()
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    lib.oracle_cell_map.argtypes = [P, P, ctypes.POINTER(_Geom), P]
    lib.oracle_cell_map.restype = ctypes.c_int64
    lib.oracle_cell_map_slabs.argtypes = [P, P, ctypes.POINTER(_Geom), ctypes.c_int32, P]
    lib.oracle_cell_map_slabs.restype = ctypes.c_int64
    lib.oracle_sort_by_cell.argtypes = [P, ctypes.c_int64, ctypes.c_int32, P, P]
    lib.oracle_sort_by_cell.restype = None
    lib.oracle_pool.argtypes = [P, P, P, ctypes.POINTER(_Geom), ctypes.c_int32,
                                ctypes.c_int32, P, P, P]
    lib.oracle_pool.restype = None
    lib.oracle_backward.argtypes = [P, P, P, P, ctypes.POINTER(_Geom), ctypes.c_int32,
                                    ctypes.c_int32, P, P]
    lib.oracle_backward.restype = None
    lib.oracle_pool_reduce.argtypes = [P, P, P, ctypes.POINTER(_Geom), ctypes.c_int32,
                                       ctypes.c_int32, ctypes.c_int32, P]
    lib.oracle_pool_reduce.restype = None
    lib.oracle_max_threads.argtypes = []
    lib.oracle_max_threads.restype = ctypes.c_int
    lib.oracle_set_threads.argtypes = [ctypes.c_int]
    lib.oracle_set_threads.restype = None
    _lib = lib
    return lib


def _geom(rig) -> _Geom:
    return _Geom(rig.n_cams, rig.feat_h, rig.feat_w, rig.n_depth,
                 rig.depth_min, rig.depth_step, rig.pixel_offset,
                 rig.nx, rig.ny, rig.x_min, rig.y_min, rig.cell_x, rig.cell_y,
                 rig.z_min, rig.z_cell)


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def cell_map(rig, nz: int = 1) -> np.ndarray:
    """int32 [N*D*H*W]: cell id of each point in point-id order, -1 if dropped.
    With nz > 1 the grid has nz stacked z slabs of z_cell each from z_min and
    the cell id is (iy * nx + ix) * nz + iz (z quantised like x and y)."""
    lib = _load()
    intr = np.ascontiguousarray(rig.intrinsics, dtype=np.float64).reshape(-1)
    extr = np.ascontiguousarray(rig.extrinsics, dtype=np.float64).reshape(-1)
    assert intr.size == 4 * rig.n_cams and extr.size == 12 * rig.n_cams and nz >= 1
    out = np.empty(rig.n_points, dtype=np.int32)
    g = _geom(rig)
    if nz == 1:
        lib.oracle_cell_map(_ptr(intr), _ptr(extr), ctypes.byref(g), _ptr(out))
    else:
        lib.oracle_cell_map_slabs(_ptr(intr), _ptr(extr), ctypes.byref(g), int(nz), _ptr(out))
    return out


def sort_by_cell(cell_of_point: np.ndarray, n_cells: int):
    """(sorted_point int32 [K], cell_start int32 [n_cells + 1])."""
    lib = _load()
    cop = np.ascontiguousarray(cell_of_point, dtype=np.int32)
    kept = int((cop >= 0).sum())
    sorted_point = np.empty(kept, dtype=np.int32)
    cell_start = np.empty(n_cells + 1, dtype=np.int32)
    lib.oracle_sort_by_cell(_ptr(cop), cop.size, n_cells, _ptr(sorted_point),
                            _ptr(cell_start))
    return sorted_point, cell_start


def plan(rig):
    """The canonical plan: (cell_of_point, sorted_point, cell_start)."""
    cop = cell_map(rig)
    sp, cs = sort_by_cell(cop, rig.n_cells)
    return cop, sp, cs


def pool(rig, cell_of_point: np.ndarray, P: np.ndarray, F: np.ndarray,
         want_f64: bool = False, want_abs: bool = False):
    """Sum pooling. P float32 [B][N][D][H][W], F float32 [B][N][H][W][C].
    Returns float32 [B][ny][nx][C]; with want_f64 / want_abs also the
    double sums and the double sums of |P * F| (in that order)."""
    lib = _load()
    P = np.ascontiguousarray(P, dtype=np.float32)
    F = np.ascontiguousarray(F, dtype=np.float32)
    B = P.shape[0]
    C = F.shape[-1]
    assert P.size == B * rig.n_points and F.size == B * rig.n_pixels * C
    cop = np.ascontiguousarray(cell_of_point, dtype=np.int32)
    out = np.empty((B, rig.ny, rig.nx, C), dtype=np.float32)
    o64 = np.empty(out.shape, dtype=np.float64) if want_f64 else None
    a64 = np.empty(out.shape, dtype=np.float64) if want_abs else None
    g = _geom(rig)
    lib.oracle_pool(_ptr(P), _ptr(F), _ptr(cop), ctypes.byref(g), B, C, _ptr(out),
                    _ptr(o64) if o64 is not None else None,
                    _ptr(a64) if a64 is not None else None)
    res = [out]
    if want_f64:
        res.append(o64)
    if want_abs:
        res.append(a64)
    return res[0] if len(res) == 1 else tuple(res)


REDUCE_MODES = {"mean": 1, "max": 2}


def pool_reduce(rig, cell_of_point: np.ndarray, P: np.ndarray, F: np.ndarray, mode: str):
    """Mean or max pooling ("Interval Reduction": mean and max are the other
    symmetric aggregations it names). Returns float64 [B][ny][nx][C]: per
    cell the mean, or the max, of P * F over its kept points; 0 for a cell
    without points."""
    lib = _load()
    P = np.ascontiguousarray(P, dtype=np.float32)
    F = np.ascontiguousarray(F, dtype=np.float32)
    B = P.shape[0]
    C = F.shape[-1]
    assert P.size == B * rig.n_points and F.size == B * rig.n_pixels * C
    cop = np.ascontiguousarray(cell_of_point, dtype=np.int32)
    out = np.empty((B, rig.ny, rig.nx, C), dtype=np.float64)
    g = _geom(rig)
    lib.oracle_pool_reduce(_ptr(P), _ptr(F), _ptr(cop), ctypes.byref(g), B, C,
                           REDUCE_MODES[mode], _ptr(out))
    return out


def slab_grid(rig, nz: int):
    """The rig with each BEV row widened to nx * nz cells, so that the cell id
    (iy * nx + ix) * nz + iz of an nz-slab cell map indexes its pooled rows,
    and [B][ny][nx * nz][C] reshapes to [B][ny][nx][nz * C]."""
    return dataclasses.replace(rig, nx=rig.nx * nz)


def plan_slabs(rig, nz: int):
    """(cell_of_point, sorted_point, cell_start) over nz stacked z slabs."""
    cop = cell_map(rig, nz)
    sp, cs = sort_by_cell(cop, rig.n_cells * nz)
    return cop, sp, cs


def pool_slabs(rig, nz: int, P: np.ndarray, F: np.ndarray, mode: str = "sum"):
    """Pooling over nz stacked z slabs, flattened along z by concatenating
    the slabs' channels (Sec. III-B: the point cloud is quantised on the grid
    and the features are flattened along the z-axis): z is quantised like x
    and y, iz = floor((z - z_min) / z_cell) in [0, nz), and
    out[b][iy][ix][iz * C + c] is the pooled value of slab iz.
    Returns float64 [B][ny][nx][nz * C]."""
    cop = cell_map(rig, nz)
    grid = slab_grid(rig, nz)
    if mode == "sum":
        out = pool(grid, cop, P, F, want_f64=True)[1]
    else:
        out = pool_reduce(grid, cop, P, F, mode)
    B, C = out.shape[0], out.shape[-1]
    return out.reshape(B, rig.ny, rig.nx, nz * C)


def backward(rig, cell_of_point: np.ndarray, P: np.ndarray, F: np.ndarray, G: np.ndarray):
    """Gradients of ``pool``. P float32 [B][N][D][H][W], F float32
    [B][N][H][W][C], G float32 [B][ny][nx][C]. Returns (dP, dF) as float64
    arrays of the shapes of P and F."""
    lib = _load()
    P = np.ascontiguousarray(P, dtype=np.float32)
    F = np.ascontiguousarray(F, dtype=np.float32)
    G = np.ascontiguousarray(G, dtype=np.float32)
    B = P.shape[0]
    C = F.shape[-1]
    assert P.size == B * rig.n_points and F.size == B * rig.n_pixels * C
    assert G.size == B * rig.n_cells * C
    cop = np.ascontiguousarray(cell_of_point, dtype=np.int32)
    dP = np.empty(P.shape, dtype=np.float64)
    dF = np.empty(F.shape, dtype=np.float64)
    g = _geom(rig)
    lib.oracle_backward(_ptr(P), _ptr(F), _ptr(G), _ptr(cop), ctypes.byref(g), B, C,
                        _ptr(dP), _ptr(dF))
    return dP, dF


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def set_threads(n: int) -> None:
    """Thread count of later oracle calls from this thread (results are
    bitwise the same for any count)."""
    _load().oracle_set_threads(int(n))
