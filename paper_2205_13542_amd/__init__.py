"""BEV pooling on MI355X: camera-fixed plan + per-frame fused lift-and-sum.

The camera-to-BEV transform of BEVFusion (arXiv 2205.13542, Sec. III-B):
each camera feature pixel is lifted to D points along its ray, each carrying
P[n,d,h,w] * F[n,h,w,:]. Every point is quantised to an r x r BEV cell, and
the points of each cell are summed. The work runs in libbevpool.so
(hand-written HIP for gfx950) behind the C ABI of include/bevpool.h. This
package is the thin binding: ``_binding`` mirrors the C calls one to one, and
``Plan`` adds torch tensor plumbing (device memory and the current stream
only). There is no CPU fallback. A missing library raises ImportError.
"""
from __future__ import annotations

import numpy as np

from . import _binding
from ._binding import (BEVPOOL_BF16, BEVPOOL_F16, BEVPOOL_F32, BEVPOOL_MAX, BEVPOOL_MEAN,
                       BEVPOOL_SUM, BevpoolError,
                       bevpool_backward, bevpool_forward, bevpool_forward_ex,
                       bevpool_forward_timed, bevpool_geometry, bevpool_to_nchw,
                       bevpool_last_error,
                       bevpool_plan, bevpool_plan_destroy, bevpool_plan_export,
                       bevpool_plan_import, bevpool_associate_noalloc, bevpool_plan_slabs,
                       bevpool_plan_info_get, bevpool_version)

__all__ = [
    "Plan", "SlabPlan", "bev_pool", "BevpoolError", "bevpool_plan", "bevpool_forward", "bevpool_forward_ex",
    "bevpool_forward_timed", "bevpool_backward", "bevpool_to_nchw", "to_nchw",
    "BEVPOOL_SUM", "BEVPOOL_MEAN", "BEVPOOL_MAX",
    "bevpool_plan_info_get",
    "bevpool_plan_export", "bevpool_plan_import", "bevpool_plan_destroy", "bevpool_last_error", "bevpool_version",
    "bevpool_geometry", "geometry_of", "BEVPOOL_F32", "BEVPOOL_BF16", "BEVPOOL_F16",
    "bevpool_associate_noalloc", "associate_noalloc", "bevpool_plan_slabs",
]

_GEOM_FIELDS = [f for f, _ in bevpool_geometry._fields_]


def geometry_of(rig) -> bevpool_geometry:
    """bevpool_geometry from any object (or mapping) with the same field names."""
    get = rig.__getitem__ if isinstance(rig, dict) else (lambda k: getattr(rig, k))
    return bevpool_geometry(*[get(f) for f in _GEOM_FIELDS])


def _torch():
    import torch
    return torch


_REDUCE = {"sum": BEVPOOL_SUM, "mean": BEVPOOL_MEAN, "max": BEVPOOL_MAX}


def _dtype_code(t) -> int:
    torch = _torch()
    codes = {torch.float32: BEVPOOL_F32, torch.bfloat16: BEVPOOL_BF16, torch.float16: BEVPOOL_F16}
    if t.dtype not in codes:
        raise BevpoolError(_binding.BEVPOOL_ERR_UNSUPPORTED_DTYPE, f"dtype {t.dtype}")
    return codes[t.dtype]


def associate_noalloc(rig, cell_of_point, sorted_point, cell_start, stream=None):
    """bevpool_associate_noalloc into caller tensors: int32 device tensors of
    n_points, n_points and nx*ny + 1 elements (contiguous). rig has the
    bevpool_geometry fields plus intrinsics and extrinsics. Allocates nothing
    on the device."""
    torch = _torch()
    geom = geometry_of(rig)
    n_points = geom.n_cams * geom.n_depth * geom.feat_h * geom.feat_w
    for t, n, name in ((cell_of_point, n_points, "cell_of_point"), (sorted_point, n_points, "sorted_point"),
                       (cell_start, geom.nx * geom.ny + 1, "cell_start")):
        if t.dtype != torch.int32 or not t.is_cuda or not t.is_contiguous() or t.numel() != n:
            raise BevpoolError(_binding.BEVPOOL_ERR_SHAPE_MISMATCH,
                               f"{name} must be a contiguous int32 device tensor of {n} elements")
    if stream is None:
        stream = torch.cuda.current_stream(cell_of_point.device)
    bevpool_associate_noalloc(rig.intrinsics, rig.extrinsics, geom, cell_of_point.data_ptr(),
                              sorted_point.data_ptr(), cell_start.data_ptr(), stream.cuda_stream)


def to_nchw(bev, out=None, stream=None):
    """fp32 device map [B][ny][nx][C] (contiguous, or a channel slice of a
    wider map) -> [B][C][ny][nx] (bevpool_to_nchw)."""
    torch = _torch()
    if bev.dim() != 4 or bev.dtype != torch.float32 or not bev.is_cuda or bev.stride(3) != 1:
        raise BevpoolError(_binding.BEVPOOL_ERR_INVALID_ARG,
                           "bev must be an fp32 device tensor [B][ny][nx][C] with unit channel stride")
    B, ny, nx, C = bev.shape
    ldi = bev.stride(2)
    if bev.stride(1) != nx * ldi or bev.stride(0) != ny * nx * ldi:
        raise BevpoolError(_binding.BEVPOOL_ERR_INVALID_ARG, "rows of bev must be evenly spaced")
    if out is None:
        out = torch.empty((B, C, ny, nx), dtype=torch.float32, device=bev.device)
    elif tuple(out.shape) != (B, C, ny, nx) or not out.is_contiguous() or out.dtype != torch.float32:
        raise BevpoolError(_binding.BEVPOOL_ERR_SHAPE_MISMATCH,
                           "out must be a contiguous fp32 tensor [B][C][ny][nx]")
    if stream is None:
        stream = torch.cuda.current_stream(bev.device)
    bevpool_to_nchw(bev.data_ptr(), ldi, out.data_ptr(), B, ny, nx, C, stream.cuda_stream)
    return out


class Plan:
    """A plan on the current HIP device (see bevpool_plan in bevpool.h).

    ``Plan(intrinsics, extrinsics, geometry)``: intrinsics [N][4] and
    extrinsics [N][12] float64 host arrays; geometry has the
    bevpool_geometry fields (e.g. a rig object or a dict).
    """

    def __init__(self, intrinsics, extrinsics, geometry, stream=None, nz: int = 1):
        torch = _torch()
        _binding.load()
        if stream is None:
            stream = torch.cuda.current_stream()
        self.geometry = geometry_of(geometry)
        intr = np.asarray(intrinsics, dtype=np.float64)
        extr = np.asarray(extrinsics, dtype=np.float64)
        if nz == 1:
            self.handle = bevpool_plan(intr, extr, self.geometry, stream.cuda_stream)
        else:
            self.handle = bevpool_plan_slabs(intr, extr, self.geometry, nz, stream.cuda_stream)
        self.info = bevpool_plan_info_get(self.handle)

    @classmethod
    def from_rig(cls, rig, stream=None, nz: int = 1) -> "Plan":
        return cls(rig.intrinsics, rig.extrinsics, rig, stream, nz=nz)

    @property
    def nz(self) -> int:
        return int(self.info.nz)

    def _rows(self, t, B, C, what):
        """A [B][ny][nx][nz * C] map of a plan with nz slabs as the library's
        rows of C floats, [B][ny][nx * nz][C] (a view; the map is contiguous)."""
        i = self.info
        if tuple(t.shape) != (B, i.ny, i.nx, i.nz * C) or not t.is_contiguous():
            raise BevpoolError(_binding.BEVPOOL_ERR_SHAPE_MISMATCH,
                               f"{what} must be a contiguous tensor [B][ny][nx][nz * C] for a plan "
                               f"with {i.nz} z slabs")
        return t.view(B, i.ny, i.nx * i.nz, C)

    @classmethod
    def from_cells(cls, cell_of_point, geometry, stream=None) -> "Plan":
        """A plan from a stored association (bevpool_plan_import):
        cell_of_point as ``export`` returns it, geometry with the
        bevpool_geometry fields."""
        torch = _torch()
        _binding.load()
        if stream is None:
            stream = torch.cuda.current_stream()
        self = cls.__new__(cls)
        self.geometry = geometry_of(geometry)
        self.handle = bevpool_plan_import(cell_of_point, self.geometry, stream.cuda_stream)
        self.info = bevpool_plan_info_get(self.handle)
        return self

    def close(self) -> None:
        if getattr(self, "handle", None):
            bevpool_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def export(self):
        """(cell_of_point, sorted_point, cell_start) as host int32 arrays."""
        i = self.info
        cop = np.empty(i.n_points, dtype=np.int32)
        sp = np.empty(i.n_kept, dtype=np.int32)
        cs = np.empty(i.n_cells + 1, dtype=np.int32)
        bevpool_plan_export(self.handle, cop, sp, cs)
        return cop, sp, cs

    def forward(self, depth_prob, cam_feat, out=None, stream=None, events=None, reduce="sum"):
        """depth_prob [B][N][D][H][W], cam_feat [B][N][H][W][C] device tensors
        of one dtype (fp32, bf16 or fp16); returns fp32 [B][ny][nx][C].
        reduce: "sum", "mean" or "max" (bevpool_forward_ex for the last two).
        out: optional fp32 [B][ny][nx][C] device tensor, contiguous or a
        channel slice of a wider map (rows out.stride(2) floats apart, the
        call then writes only that slice).
        events: optional (start, stop) pair of timing-enabled torch.cuda.Event,
        recorded by the forward's own first and last kernel dispatch
        (bevpool_forward_timed; sum only)."""
        torch = _torch()
        i = self.info
        if depth_prob.dim() != 5 or cam_feat.dim() != 5:
            raise BevpoolError(_binding.BEVPOOL_ERR_SHAPE_MISMATCH,
                               "depth_prob and cam_feat must be 5-D")
        B, C = depth_prob.shape[0], cam_feat.shape[-1]
        if tuple(depth_prob.shape) != (B, i.n_cams, i.n_depth, i.feat_h, i.feat_w):
            raise BevpoolError(_binding.BEVPOOL_ERR_SHAPE_MISMATCH,
                               f"depth_prob shape {tuple(depth_prob.shape)} does not match the plan")
        if tuple(cam_feat.shape) != (B, i.n_cams, i.feat_h, i.feat_w, C):
            raise BevpoolError(_binding.BEVPOOL_ERR_SHAPE_MISMATCH,
                               f"cam_feat shape {tuple(cam_feat.shape)} does not match the plan")
        if cam_feat.dtype != depth_prob.dtype:
            raise BevpoolError(_binding.BEVPOOL_ERR_UNSUPPORTED_DTYPE,
                               "depth_prob and cam_feat must share a dtype")
        if not (depth_prob.is_cuda and cam_feat.is_cuda):
            raise BevpoolError(_binding.BEVPOOL_ERR_INVALID_ARG, "inputs must be device tensors")
        if not (depth_prob.is_contiguous() and cam_feat.is_contiguous()):
            raise BevpoolError(_binding.BEVPOOL_ERR_INVALID_ARG, "inputs must be contiguous")
        if reduce not in _REDUCE:
            raise BevpoolError(_binding.BEVPOOL_ERR_INVALID_ARG, f"reduce {reduce!r}")
        nx = i.nx * i.nz
        if out is None:
            out = torch.empty((B, i.ny, i.nx, i.nz * C), dtype=torch.float32, device=cam_feat.device)
        result = out
        if i.nz > 1:
            out = self._rows(out, B, C, "out")
        ldo = out.stride(2) if out.dim() == 4 else -1
        if (tuple(out.shape) != (B, i.ny, nx, C) or out.dtype != torch.float32
                or not out.is_cuda or out.stride(3) != 1 or ldo < C
                or out.stride(1) != nx * ldo or out.stride(0) != i.ny * nx * ldo):
            raise BevpoolError(_binding.BEVPOOL_ERR_SHAPE_MISMATCH,
                               "out must be an fp32 device tensor [B][ny][nx][C] whose rows are "
                               "evenly spaced (contiguous, or a channel slice of a wider map)")
        if stream is None:
            stream = torch.cuda.current_stream(cam_feat.device)
        if reduce != "sum" or ldo != C:
            if events is not None:
                raise BevpoolError(_binding.BEVPOOL_ERR_INVALID_ARG,
                                   "timing events go with a plain sum into a contiguous map")
            bevpool_forward_ex(depth_prob.data_ptr(), cam_feat.data_ptr(), self.handle,
                               out.data_ptr(), ldo, B, C, _dtype_code(cam_feat), _REDUCE[reduce],
                               stream.cuda_stream)
        elif events is None:
            bevpool_forward(depth_prob.data_ptr(), cam_feat.data_ptr(), self.handle,
                            out.data_ptr(), B, C, _dtype_code(cam_feat), stream.cuda_stream)
        else:
            start, stop = events
            for e in (start, stop):
                if e.cuda_event == 0:       # torch creates the HIP event on first record
                    e.record(stream)
            bevpool_forward_timed(depth_prob.data_ptr(), cam_feat.data_ptr(), self.handle,
                                  out.data_ptr(), B, C, _dtype_code(cam_feat), stream.cuda_stream,
                                  start.cuda_event, stop.cuda_event)
        return result

    def backward(self, grad_out, depth_prob, cam_feat, want_depth=True, want_feat=True,
                 stream=None):
        """Gradients of forward: grad_out fp32 [B][ny][nx][C] and the forward's
        inputs; returns (grad_depth fp32 [B][N][D][H][W] or None,
        grad_feat fp32 [B][N][H][W][C] or None)."""
        torch = _torch()
        i = self.info
        B, C = depth_prob.shape[0], cam_feat.shape[-1]
        if (tuple(depth_prob.shape) != (B, i.n_cams, i.n_depth, i.feat_h, i.feat_w)
                or tuple(cam_feat.shape) != (B, i.n_cams, i.feat_h, i.feat_w, C)
                or tuple(grad_out.shape) != (B, i.ny, i.nx, i.nz * C)):
            raise BevpoolError(_binding.BEVPOOL_ERR_SHAPE_MISMATCH,
                               "grad_out, depth_prob or cam_feat does not match the plan")
        if cam_feat.dtype != depth_prob.dtype or grad_out.dtype != torch.float32:
            raise BevpoolError(_binding.BEVPOOL_ERR_UNSUPPORTED_DTYPE,
                               "depth_prob and cam_feat must share a dtype; grad_out is fp32")
        for t in (grad_out, depth_prob, cam_feat):
            if not (t.is_cuda and t.is_contiguous()):
                raise BevpoolError(_binding.BEVPOOL_ERR_INVALID_ARG,
                                   "inputs must be contiguous device tensors")
        dev = cam_feat.device
        gd = torch.empty(tuple(depth_prob.shape), dtype=torch.float32, device=dev) if want_depth else None
        gf = torch.empty(tuple(cam_feat.shape), dtype=torch.float32, device=dev) if want_feat else None
        if stream is None:
            stream = torch.cuda.current_stream(dev)
        bevpool_backward(grad_out.data_ptr(), depth_prob.data_ptr(), cam_feat.data_ptr(),
                         self.handle, gd.data_ptr() if gd is not None else 0,
                         gf.data_ptr() if gf is not None else 0, B, C, _dtype_code(cam_feat),
                         stream.cuda_stream)
        return gd, gf


class SlabPlan(Plan):
    """A plan over nz stacked z slabs, flattened along z by concatenating
    their channels (Sec. III-B, first paragraph: the lifted points are
    quantised on the grid, z like x and y, and the features flattened along
    the z-axis). Slab iz is [z_min + iz z_cell, z_min + (iz+1) z_cell);
    forward returns one [B][ny][nx][nz * C] map, channel iz * C + c being
    channel c of slab iz, from a single library call that reads P and F
    once (bevpool_plan_slabs: one association over nx * ny * nz cells)."""

    def __init__(self, intrinsics, extrinsics, geometry, nz: int, stream=None):
        if nz < 1:
            raise BevpoolError(_binding.BEVPOOL_ERR_INVALID_ARG, f"nz={nz} must be >= 1")
        super().__init__(intrinsics, extrinsics, geometry, stream, nz=nz)

    @classmethod
    def from_rig(cls, rig, nz: int, stream=None) -> "SlabPlan":
        return cls(rig.intrinsics, rig.extrinsics, rig, nz, stream)


def _autograd_function():
    torch = _torch()

    class _BevPool(torch.autograd.Function):
        """Sum pooling with its gradients (bevpool_forward, bevpool_backward)."""

        @staticmethod
        def forward(ctx, depth_prob, cam_feat, plan):
            ctx.plan = plan
            ctx.save_for_backward(depth_prob, cam_feat)
            return plan.forward(depth_prob, cam_feat)

        @staticmethod
        def backward(ctx, grad_out):
            depth_prob, cam_feat = ctx.saved_tensors
            gd, gf = ctx.plan.backward(grad_out.contiguous(), depth_prob, cam_feat,
                                       want_depth=ctx.needs_input_grad[0],
                                       want_feat=ctx.needs_input_grad[1])
            if gd is not None and gd.dtype != depth_prob.dtype:
                gd = gd.to(depth_prob.dtype)
            if gf is not None and gf.dtype != cam_feat.dtype:
                gf = gf.to(cam_feat.dtype)
            return gd, gf, None

    return _BevPool


_BEVPOOL_FN = None


def bev_pool(depth_prob, cam_feat, plan):
    """Differentiable sum pooling for training: the BEV map [B][ny][nx][C]
    fp32 of ``plan.forward``, whose gradients with respect to depth_prob and
    cam_feat come from ``plan.backward`` (returned in the inputs' dtypes)."""
    global _BEVPOOL_FN
    if _BEVPOOL_FN is None:
        _BEVPOOL_FN = _autograd_function()
    return _BEVPOOL_FN.apply(depth_prob, cam_feat, plan)
