"""ctypes binding of libbevpool.so: the C ABI of include/bevpool.h under the
same names, with argument marshalling only. Every step of the pooling runs in
the library's HIP kernels; nothing here computes.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libbevpool.so")

BEVPOOL_OK = 0
BEVPOOL_ERR_INVALID_ARG = -1
BEVPOOL_ERR_SHAPE_MISMATCH = -2
BEVPOOL_ERR_UNSUPPORTED_DTYPE = -3
BEVPOOL_ERR_OVERFLOW = -4
BEVPOOL_ERR_OOM = -5
BEVPOOL_ERR_HIP = -6

BEVPOOL_F32, BEVPOOL_BF16, BEVPOOL_F16 = 0, 1, 2
BEVPOOL_SUM, BEVPOOL_MEAN, BEVPOOL_MAX = 0, 1, 2

EXPORTED = ("bevpool_plan", "bevpool_forward", "bevpool_forward_ex", "bevpool_forward_timed",
            "bevpool_backward", "bevpool_to_nchw", "bevpool_plan_import",
            "bevpool_plan_info_get",
            "bevpool_plan_export", "bevpool_plan_destroy", "bevpool_last_error",
            "bevpool_version", "bevpool_associate_noalloc", "bevpool_plan_slabs")


class BevpoolError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"bevpool error {code}: {message}")
        self.code = code


class bevpool_geometry(ctypes.Structure):
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


class bevpool_plan_info(ctypes.Structure):
    _fields_ = [
        ("n_points", ctypes.c_int64), ("n_kept", ctypes.c_int64),
        ("n_cells", ctypes.c_int32), ("n_nonempty", ctypes.c_int32),
        ("max_per_cell", ctypes.c_int32),
        ("n_cams", ctypes.c_int32), ("n_depth", ctypes.c_int32),
        ("feat_h", ctypes.c_int32), ("feat_w", ctypes.c_int32),
        ("nx", ctypes.c_int32), ("ny", ctypes.c_int32),
        ("n_column", ctypes.c_int32), ("n_generic", ctypes.c_int32),
        ("n_empty", ctypes.c_int32), ("n_runs", ctypes.c_int32),
        ("n_partials", ctypes.c_int32), ("n_multi", ctypes.c_int32),
        ("nz", ctypes.c_int32), ("n_planes", ctypes.c_int32),
    ]


_lib = None


def load(path: str = LIB_PATH):
    """Load the library; raises (never falls back) if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"libbevpool.so is not built ({path}); run "
                          "`python -m paper_2205_13542_amd.build` first")
    lib = ctypes.CDLL(path)
    vp, i32, dp = ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER(ctypes.c_double)
    lib.bevpool_plan.argtypes = [dp, dp, ctypes.POINTER(bevpool_geometry), vp,
                                 ctypes.POINTER(vp)]
    lib.bevpool_plan.restype = ctypes.c_int
    lib.bevpool_plan_slabs.argtypes = [dp, dp, ctypes.POINTER(bevpool_geometry), i32, vp,
                                       ctypes.POINTER(vp)]
    lib.bevpool_plan_slabs.restype = ctypes.c_int
    lib.bevpool_forward.argtypes = [vp, vp, vp, vp, i32, i32, i32, vp]
    lib.bevpool_forward.restype = ctypes.c_int
    lib.bevpool_forward_ex.argtypes = [vp, vp, vp, vp, ctypes.c_int64, i32, i32, i32, i32, vp]
    lib.bevpool_forward_ex.restype = ctypes.c_int
    lib.bevpool_plan_import.argtypes = [vp, ctypes.POINTER(bevpool_geometry), vp,
                                        ctypes.POINTER(ctypes.c_void_p)]
    lib.bevpool_plan_import.restype = ctypes.c_int
    lib.bevpool_to_nchw.argtypes = [vp, ctypes.c_int64, vp, i32, i32, i32, i32, vp]
    lib.bevpool_to_nchw.restype = ctypes.c_int
    lib.bevpool_forward_timed.argtypes = [vp, vp, vp, vp, i32, i32, i32, vp, vp, vp]
    lib.bevpool_forward_timed.restype = ctypes.c_int
    lib.bevpool_backward.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, vp]
    lib.bevpool_backward.restype = ctypes.c_int
    lib.bevpool_plan_info_get.argtypes = [vp, ctypes.POINTER(bevpool_plan_info)]
    lib.bevpool_plan_info_get.restype = ctypes.c_int
    lib.bevpool_plan_export.argtypes = [vp, vp, vp, vp]
    lib.bevpool_plan_export.restype = ctypes.c_int
    lib.bevpool_plan_destroy.argtypes = [vp]
    lib.bevpool_plan_destroy.restype = None
    lib.bevpool_last_error.argtypes = []
    lib.bevpool_last_error.restype = ctypes.c_char_p
    lib.bevpool_associate_noalloc.argtypes = [dp, dp, ctypes.POINTER(bevpool_geometry), vp, vp, vp, vp]
    lib.bevpool_associate_noalloc.restype = ctypes.c_int
    lib.bevpool_version.argtypes = []
    lib.bevpool_version.restype = ctypes.c_int32
    _lib = lib
    return lib


def _check(rc: int) -> None:
    if rc != BEVPOOL_OK:
        msg = load().bevpool_last_error().decode(errors="replace")
        raise BevpoolError(rc, msg)


def bevpool_last_error() -> str:
    return load().bevpool_last_error().decode(errors="replace")


def bevpool_version() -> int:
    return int(load().bevpool_version())


def bevpool_plan(intrinsics, extrinsics, geom: bevpool_geometry, hip_stream: int = 0) -> int:
    """intrinsics / extrinsics: host float64 buffers (numpy arrays or ctypes
    arrays) of n_cams*4 and n_cams*12 values. Returns the plan handle."""
    import numpy as np
    intr = np.ascontiguousarray(intrinsics, dtype=np.float64).reshape(-1)
    extr = np.ascontiguousarray(extrinsics, dtype=np.float64).reshape(-1)
    out = ctypes.c_void_p()
    dp = ctypes.POINTER(ctypes.c_double)
    _check(load().bevpool_plan(intr.ctypes.data_as(dp), extr.ctypes.data_as(dp),
                               ctypes.byref(geom), ctypes.c_void_p(hip_stream),
                               ctypes.byref(out)))
    return int(out.value)


def bevpool_plan_slabs(intrinsics, extrinsics, geom: bevpool_geometry, nz: int,
                       hip_stream: int = 0) -> int:
    """A plan over nz stacked z slabs; returns the plan handle."""
    import numpy as np
    intr = np.ascontiguousarray(intrinsics, dtype=np.float64).reshape(-1)
    extr = np.ascontiguousarray(extrinsics, dtype=np.float64).reshape(-1)
    out = ctypes.c_void_p()
    dp = ctypes.POINTER(ctypes.c_double)
    _check(load().bevpool_plan_slabs(intr.ctypes.data_as(dp), extr.ctypes.data_as(dp),
                                     ctypes.byref(geom), int(nz), ctypes.c_void_p(hip_stream),
                                     ctypes.byref(out)))
    return int(out.value)


def bevpool_associate_noalloc(intrinsics, extrinsics, geom: bevpool_geometry, cell_of_point: int,
                              sorted_point: int, cell_start: int, hip_stream: int = 0) -> None:
    """intrinsics / extrinsics: host float64 arrays; the three outputs are
    device pointers (int32 [n_points], [n_points], [nx*ny + 1])."""
    import numpy as np
    intr = np.ascontiguousarray(intrinsics, dtype=np.float64).reshape(-1)
    extr = np.ascontiguousarray(extrinsics, dtype=np.float64).reshape(-1)
    dp = ctypes.POINTER(ctypes.c_double)
    _check(load().bevpool_associate_noalloc(intr.ctypes.data_as(dp), extr.ctypes.data_as(dp),
                                            ctypes.byref(geom), ctypes.c_void_p(cell_of_point),
                                            ctypes.c_void_p(sorted_point), ctypes.c_void_p(cell_start),
                                            ctypes.c_void_p(hip_stream)))


def bevpool_plan_import(cell_of_point, geom: bevpool_geometry, hip_stream: int = 0) -> int:
    """cell_of_point: host int32 array [n_points] (as exported)."""
    import numpy as np
    cop = np.ascontiguousarray(cell_of_point, dtype=np.int32)
    out = ctypes.c_void_p()
    _check(load().bevpool_plan_import(cop.ctypes.data_as(ctypes.c_void_p), ctypes.byref(geom),
                                      ctypes.c_void_p(hip_stream), ctypes.byref(out)))
    return int(out.value)


def bevpool_forward(depth_prob: int, cam_feat: int, plan: int, bev_out: int,
                    batch: int, channels: int, dtype: int, hip_stream: int = 0) -> None:
    """All buffers are device addresses (ints)."""
    _check(load().bevpool_forward(ctypes.c_void_p(depth_prob), ctypes.c_void_p(cam_feat),
                                  ctypes.c_void_p(plan), ctypes.c_void_p(bev_out),
                                  batch, channels, dtype, ctypes.c_void_p(hip_stream)))


def bevpool_forward_ex(depth_prob: int, cam_feat: int, plan: int, bev_out: int,
                       out_row_stride: int, batch: int, channels: int, dtype: int, reduce: int,
                       hip_stream: int = 0) -> None:
    """bevpool_forward with an aggregation (BEVPOOL_SUM, _MEAN, _MAX) and an
    output row stride in floats; device addresses as ints."""
    _check(load().bevpool_forward_ex(ctypes.c_void_p(depth_prob), ctypes.c_void_p(cam_feat),
                                     ctypes.c_void_p(plan), ctypes.c_void_p(bev_out),
                                     out_row_stride, batch, channels, dtype, reduce,
                                     ctypes.c_void_p(hip_stream)))


def bevpool_to_nchw(bev_nhwc: int, in_row_stride: int, bev_nchw: int, batch: int, ny: int,
                    nx: int, channels: int, hip_stream: int = 0) -> None:
    """Rows [B][ny*nx] (in_row_stride floats apart) to planes [B][C][ny][nx];
    device addresses as ints."""
    _check(load().bevpool_to_nchw(ctypes.c_void_p(bev_nhwc), in_row_stride,
                                  ctypes.c_void_p(bev_nchw), batch, ny, nx, channels,
                                  ctypes.c_void_p(hip_stream)))


def bevpool_forward_timed(depth_prob: int, cam_feat: int, plan: int, bev_out: int, batch: int,
                          channels: int, dtype: int, hip_stream: int, start_event: int,
                          stop_event: int) -> None:
    """bevpool_forward with kernel-boundary events (hipEvent_t handles as
    ints; 0 for none)."""
    _check(load().bevpool_forward_timed(ctypes.c_void_p(depth_prob), ctypes.c_void_p(cam_feat),
                                        ctypes.c_void_p(plan), ctypes.c_void_p(bev_out),
                                        batch, channels, dtype, ctypes.c_void_p(hip_stream),
                                        ctypes.c_void_p(start_event), ctypes.c_void_p(stop_event)))


def bevpool_backward(grad_out: int, depth_prob: int, cam_feat: int, plan: int, grad_depth: int,
                     grad_feat: int, batch: int, channels: int, dtype: int,
                     hip_stream: int = 0) -> None:
    """Device addresses as ints; grad_depth or grad_feat may be 0 (skip)."""
    _check(load().bevpool_backward(ctypes.c_void_p(grad_out), ctypes.c_void_p(depth_prob),
                                   ctypes.c_void_p(cam_feat), ctypes.c_void_p(plan),
                                   ctypes.c_void_p(grad_depth or None),
                                   ctypes.c_void_p(grad_feat or None), batch, channels, dtype,
                                   ctypes.c_void_p(hip_stream)))


def bevpool_plan_info_get(plan: int) -> bevpool_plan_info:
    info = bevpool_plan_info()
    _check(load().bevpool_plan_info_get(ctypes.c_void_p(plan), ctypes.byref(info)))
    return info


def bevpool_plan_export(plan: int, cell_of_point=None, sorted_point=None, cell_start=None) -> None:
    """Copy into host int32 numpy arrays (any may be None)."""
    def ptr(a):
        return None if a is None else ctypes.c_void_p(a.ctypes.data)
    _check(load().bevpool_plan_export(ctypes.c_void_p(plan), ptr(cell_of_point),
                                      ptr(sorted_point), ptr(cell_start)))


def bevpool_plan_destroy(plan: int) -> None:
    load().bevpool_plan_destroy(ctypes.c_void_p(plan))
