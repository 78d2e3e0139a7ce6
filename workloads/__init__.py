"""Seeded synthetic workloads for BEV pooling: camera rigs and per-frame inputs.

This module only draws inputs. It holds none of the pooling arithmetic
(projection, quantisation, sorting, reduction), so both the oracle side and
the GPU side of a test can take their inputs from here.

A workload is a camera rig (intrinsics, extrinsics, frustum and BEV grid) plus
per-frame depth probabilities P[B][N][D][H][W] and camera features
F[B][N][H][W][C], the two inputs of the camera-to-BEV transform (BEVFusion,
Sec. III-B, first paragraph). Sizes follow the paper's typical workload
(six cameras, 32x88 feature maps from 256x704 images at stride 8, depth
1-60 m at 0.5 m: Sec. III-B, second paragraph and its footnote). The data are
synthetic stand-ins for nuScenes: no images, trained depth network or dataset
records are used.

Reduced-precision inputs are returned as float32 arrays whose values are
already rounded (round-to-nearest-even) to bf16 or fp16, so they widen back
exactly; ``dtype`` says which format the device copy uses.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

__all__ = [
    "Rig", "Workload", "tiny_rig", "identity_rig", "ring_rig", "tilt_rig",
    "round_bf16", "round_f16", "make", "WORKLOADS",
]


@dataclasses.dataclass(frozen=True)
class Rig:
    """Camera rig, frustum and BEV grid.

    intrinsics: float64 [N][4] = fx, fy, cx, cy in feature-grid pixels.
    extrinsics: float64 [N][12] = row-major [R | t], camera frame to ego frame.
    Camera axes: x right, y down, z forward. Ego axes: x forward, y left, z up.
    Depth bin k sits at depth_min + k * depth_step; pixel (h, w) at
    (w + pixel_offset, h + pixel_offset). The grid covers
    [x_min, x_min + nx*cell_x) x [y_min, y_min + ny*cell_y) and one z slab
    [z_min, z_min + z_cell).
    """
    n_cams: int
    feat_h: int
    feat_w: int
    n_depth: int
    depth_min: float
    depth_step: float
    pixel_offset: float
    nx: int
    ny: int
    x_min: float
    y_min: float
    cell_x: float
    cell_y: float
    z_min: float
    z_cell: float
    intrinsics: np.ndarray
    extrinsics: np.ndarray

    @property
    def n_points(self) -> int:
        return self.n_cams * self.n_depth * self.feat_h * self.feat_w

    @property
    def n_cells(self) -> int:
        return self.nx * self.ny

    @property
    def n_pixels(self) -> int:
        return self.n_cams * self.feat_h * self.feat_w


@dataclasses.dataclass
class Workload:
    name: str
    rig: Rig
    channels: int
    batch: int
    dtype: str           # "f32", "bf16" or "f16": the device input format
    P: np.ndarray        # float32 [B][N][D][H][W]
    F: np.ndarray        # float32 [B][N][H][W][C]


# ---------------------------------------------------------------- rigs

def tiny_rig() -> Rig:
    """One camera at the ego origin looking along ego +x; 4x8 features,
    8 depth bins at 1..8 m, fx=fy=4, cx=4, cy=2; 16x16 cells of 1 m over
    [-8, 8)^2; z slab [-10, 10)."""
    R = np.array([[0.0, 0.0, 1.0],
                  [-1.0, 0.0, 0.0],
                  [0.0, -1.0, 0.0]])
    E = np.concatenate([R, np.zeros((3, 1))], axis=1).reshape(1, 12)
    return Rig(1, 4, 8, 8, 1.0, 1.0, 0.5, 16, 16, -8.0, -8.0, 1.0, 1.0,
               -10.0, 20.0, np.array([[4.0, 4.0, 4.0, 2.0]]), E.copy())


def identity_rig() -> Rig:
    """The tiny rig with identity extrinsics: the camera looks along ego +z,
    so every point lies inside the [-8, 8)^2 grid and the z slab."""
    r = tiny_rig()
    E = np.concatenate([np.eye(3), np.zeros((3, 1))], axis=1).reshape(1, 12)
    return dataclasses.replace(r, extrinsics=E)


def _ring_extrinsics(n_cams: int, radius: float, height: float) -> np.ndarray:
    """Cameras on a ring at yaw 360/n_cams * k, facing outward, level."""
    E = np.zeros((n_cams, 12))
    for k in range(n_cams):
        psi = math.radians(360.0 / n_cams * k)
        s, c = math.sin(psi), math.cos(psi)
        R = np.array([[s, 0.0, c],
                      [-c, 0.0, s],
                      [0.0, -1.0, 0.0]])
        t = np.array([radius * c, radius * s, height])
        E[k] = np.concatenate([R, t[:, None]], axis=1).reshape(12)
    return E


def ring_rig(scale: int = 1) -> Rig:
    """nuScenes-shaped rig: six cameras at 60 degree yaw spacing on a ring of
    radius 1 m at height 1.5 m; images 256x704 at stride 8 (32x88 features),
    fx=fy=560 px at image scale; depth 1-60 m at 0.5 m (118 bins); BEV
    360x360 at 0.3 m over [-54, 54)^2. ``scale=2`` is the high-resolution
    variant: 512x1408 images (64x176 features), 236 bins at 0.25 m, and a
    720x720 grid at 0.15 m."""
    H, W = 32 * scale, 88 * scale
    f = 70.0 * scale
    intr = np.tile(np.array([[f, f, W / 2.0, H / 2.0]]), (6, 1))
    return Rig(6, H, W, 118 * scale, 1.0, 0.5 / scale, 0.5,
               360 * scale, 360 * scale, -54.0, -54.0, 0.3 / scale, 0.3 / scale,
               -10.0, 20.0, intr, _ring_extrinsics(6, 1.0, 1.5))


def tilt_rig(rig: Rig, pitch_deg: float = 5.0, roll_deg: float = 2.0) -> Rig:
    """Every camera pitched about its x axis and rolled about its z axis, so
    a point's cell depends on its pixel row as well as its column."""
    a, b = math.radians(pitch_deg), math.radians(roll_deg)
    pitch = np.array([[1.0, 0.0, 0.0],
                      [0.0, math.cos(a), -math.sin(a)],
                      [0.0, math.sin(a), math.cos(a)]])
    roll = np.array([[math.cos(b), -math.sin(b), 0.0],
                     [math.sin(b), math.cos(b), 0.0],
                     [0.0, 0.0, 1.0]])
    E = rig.extrinsics.copy().reshape(-1, 3, 4)
    for k in range(E.shape[0]):
        E[k, :, :3] = E[k, :, :3] @ pitch @ roll
    return dataclasses.replace(rig, extrinsics=E.reshape(-1, 12))


# ---------------------------------------------------------------- inputs

def _softmax_depth(logits: np.ndarray) -> np.ndarray:
    """Softmax over the depth axis (axis 1 of [N][D][H][W]) in float64,
    rounded to float32."""
    z = logits - logits.max(axis=1, keepdims=True)
    e = np.exp(z)
    return (e / e.sum(axis=1, keepdims=True)).astype(np.float32)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even), kept as float32."""
    bits = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    bits = (bits + 0x7FFF + ((bits >> 16) & 1)) & 0xFFFF0000
    return bits.astype(np.uint32).view(np.float32)


def round_f16(x: np.ndarray) -> np.ndarray:
    return np.asarray(x, dtype=np.float32).astype(np.float16).astype(np.float32)


def depth_normal_softmax(rng, rig: Rig) -> np.ndarray:
    """Softmax over depth of N(0,1) logits."""
    shape = (rig.n_cams, rig.n_depth, rig.feat_h, rig.feat_w)
    return _softmax_depth(rng.standard_normal(shape))


def depth_gaussian_peaked(rng, rig: Rig, sigma_bins: float = 3.0,
                          noise: float = 0.5) -> np.ndarray:
    """Per pixel a peak at a uniform random bin mu: logits
    -(k - mu)^2 / (2 sigma^2) + N(0, noise^2), softmaxed over depth."""
    N, D, H, W = rig.n_cams, rig.n_depth, rig.feat_h, rig.feat_w
    mu = rng.integers(0, D, size=(N, 1, H, W))
    k = np.arange(D, dtype=np.float64).reshape(1, D, 1, 1)
    logits = -((k - mu) ** 2) / (2.0 * sigma_bins ** 2)
    logits = logits + rng.normal(0.0, noise, size=(N, D, H, W))
    return _softmax_depth(logits)


def depth_sparse(rng, rig: Rig, p_onehot: float = 0.9) -> np.ndarray:
    """90% of pixels one-hot at a uniform bin, the rest a softmax of N(0,1)
    logits: most depth probabilities are exactly zero."""
    N, D, H, W = rig.n_cams, rig.n_depth, rig.feat_h, rig.feat_w
    onehot_bin = rng.integers(0, D, size=(N, H, W))
    is_onehot = rng.random(size=(N, H, W)) < p_onehot
    soft = _softmax_depth(rng.standard_normal((N, D, H, W)))
    hot = (np.arange(D).reshape(1, D, 1, 1) == onehot_bin[:, None]).astype(np.float32)
    return np.where(is_onehot[:, None], hot, soft).astype(np.float32)


def features_normal(rng, rig: Rig, channels: int) -> np.ndarray:
    shape = (rig.n_cams, rig.feat_h, rig.feat_w, channels)
    return rng.standard_normal(shape).astype(np.float32)


_DEPTH = {
    "normal": depth_normal_softmax,
    "peaked": depth_gaussian_peaked,
    "sparse": depth_sparse,
}


def frames(rig: Rig, channels: int, batch: int, depth: str, seed: int,
           dtype: str = "f32"):
    """Draw ``batch`` frames; frame b uses seed ``seed + b``. For each frame
    the depth draw comes first, then the features. Returns (P, F) float32."""
    Ps, Fs = [], []
    for b in range(batch):
        rng = np.random.default_rng(seed + b)
        Ps.append(_DEPTH[depth](rng, rig))
        Fs.append(features_normal(rng, rig, channels))
    P, F = np.stack(Ps), np.stack(Fs)
    if dtype == "bf16":
        P, F = round_bf16(P), round_bf16(F)
    elif dtype == "f16":
        P, F = round_f16(P), round_f16(F)
    elif dtype != "f32":
        raise ValueError(f"unknown dtype {dtype!r}")
    return P, F


# name -> (rig factory, channels, batch, depth generator, dtype)
WORKLOADS = {
    # 1 camera, 4x8 features, 8 bins, C=8 -> 16x16 cells
    "tiny": (tiny_rig, 8, 1, "normal", "f32"),
    # 6 cameras x 118 bins x 32x88, C=80 fp32 -> 360x360 cells
    "nuscenes": (ring_rig, 80, 1, "peaked", "f32"),
    # the same frame with bf16 / fp16 inputs, fp32 accumulation and output
    "nuscenes_bf16": (ring_rig, 80, 1, "peaked", "bf16"),
    "nuscenes_f16": (ring_rig, 80, 1, "peaked", "f16"),
    # 8 independent frames sharing one plan
    "nuscenes_b8": (ring_rig, 80, 8, "peaked", "f32"),
    # 6 cameras x 236 bins x 64x176, C=128 -> 720x720 cells, sparse depth
    "highres": (lambda: ring_rig(2), 128, 1, "sparse", "f32"),
    # test-only rigs
    "tiny_identity": (identity_rig, 8, 1, "normal", "f32"),
    "nuscenes_tilted": (lambda: tilt_rig(ring_rig()), 80, 1, "peaked", "f32"),
    # the same rig with a calibration-sized tilt: pitch 1 deg, roll 0.5 deg
    "nuscenes_tilt1": (lambda: tilt_rig(ring_rig(), 1.0, 0.5), 80, 1, "peaked", "f32"),
}


def make(name: str, seed: int = 0, batch: int | None = None,
         channels: int | None = None) -> Workload:
    factory, C, B, depth, dtype = WORKLOADS[name]
    rig = factory()
    C = C if channels is None else channels
    B = B if batch is None else batch
    P, F = frames(rig, C, B, depth, seed, dtype)
    return Workload(name, rig, C, B, dtype, P, F)
