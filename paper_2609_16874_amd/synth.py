"""Seeded synthetic frames for the centroid-encoding decoder.

This module only *draws inputs*: instance shapes, the target encoding of
each instance's centroid (the paper's Eq1 with Eq2's sin/cos pairs, here
with per-axis angular frequencies in radians per pixel), Gaussian noise and
the foreground channel.  It contains none of the decoding arithmetic and is
shared, unchanged, by the tests, the benchmark and the oracle's callers.

Frame recipe (all draws from one ``numpy.random.Generator(PCG64)`` seeded
with ``SeedSequence([260916874, config, *extra])``, in this order):

1. instances, one after another (shape kind, centre, size, shape params);
   rasterised on pixel centres (j+0.5, i+0.5) into an int32 instance map,
   later instances overwriting earlier ones;
2. centroid of every instance = fp64 mean of its *visible* pixel centres
   (instances left with no pixel are dropped);
3. optional outlier pixels (uniform, without replacement) whose clean
   embedding encodes a uniformly random position instead;
4. embedding = clean encoding (0 on background) + N(0, sigma^2) per channel,
   drawn as float32;
5. foreground channel = 1{instance} + N(0, 0.05^2), drawn as float32;
6. both cast to the frame dtype (round to nearest even).

Channel layout per pixel (channels-last ``[H][W][D]``, ``D = 4F``): the
x block (channels ``0..2F-1``) then the y block (``2F..4F-1``); inside a
block harmonic ``k`` occupies ``(2k, 2k+1) = (sin, cos)``.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

SEED_BASE = 260916874


@dataclass(frozen=True)
class FrameSpec:
    """Shape and statistics of one synthetic workload."""

    name: str
    H: int
    W: int
    n_freq: int               # harmonics per axis (F); D = 4F
    dtype: str                # "f32" or "f16"
    period_x: float           # base period (pixels) of harmonic 0 along x
    period_y: float
    sigma: float              # embedding noise std
    fg_sigma: float = 0.05    # foreground-channel noise std
    outlier_frac: float = 0.0
    n_frames: int = 1
    bins: int = 32
    fg_threshold: float = 0.5
    # instance recipe
    kind: str = "mixed"       # "ellipse", "polygon" or "mixed"
    n_inst: tuple = (4, 4)    # inclusive range of the instance count
    radius: tuple = (10.0, 120.0)
    radius_law: str = "loguniform"   # "uniform", "loguniform", "semi" or "rowdep"

    @property
    def D(self) -> int:
        return 4 * self.n_freq

    @property
    def np_dtype(self):
        return np.float32 if self.dtype == "f32" else np.float16

    def freqs(self):
        """Angular frequencies (rad/px) of the geometric harmonic ladder."""
        fx = np.array([2.0 * math.pi * (2.0 ** k) / self.period_x for k in range(self.n_freq)])
        fy = np.array([2.0 * math.pi * (2.0 ** k) / self.period_y for k in range(self.n_freq)])
        return fx, fy

    def emb_bytes(self) -> int:
        return self.H * self.W * self.D * np.dtype(self.np_dtype).itemsize


# The five workloads.  Sizes, shapes, noise and frequency ladders follow the
# workload descriptions; where a base period is not given it is the axis
# extent (each axis is normalised on its own).
CONFIGS = {
    0: FrameSpec("64x64 D32 f32 4 ellipses", 64, 64, 8, "f32", 64.0, 64.0, 0.05,
                 kind="ellipse", n_inst=(4, 4), radius=(6.0, 16.0), radius_law="semi"),
    1: FrameSpec("256x256 D32 f32 20 polygons", 256, 256, 8, "f32", 256.0, 256.0, 0.1,
                 kind="polygon", n_inst=(20, 20), radius=(8.0, 40.0), radius_law="uniform"),
    2: FrameSpec("640x640 D64 f16 50 mixed +1% outliers", 640, 640, 16, "f16", 640.0, 640.0, 0.1,
                 outlier_frac=0.01, kind="mixed", n_inst=(50, 50), radius=(10.0, 120.0)),
    3: FrameSpec("1024x2048 D64 f16 150 mixed row-dependent", 1024, 2048, 16, "f16", 2048.0, 1024.0, 0.15,
                 kind="mixed", n_inst=(150, 150), radius=(4.0, 200.0), radius_law="rowdep"),
    4: FrameSpec("16x 640x640 D64 f16 10-100 mixed", 640, 640, 16, "f16", 640.0, 640.0, 0.1,
                 n_frames=16, kind="mixed", n_inst=(10, 100), radius=(10.0, 120.0)),
    # the paper's own decoder shape: 616x616 input -> 704x704 maps, L = 4
    # harmonics per axis (D = 16) in fp32; used for the bin-count sweep
    5: FrameSpec("704x704 D16 f32 50 mixed", 704, 704, 4, "f32", 704.0, 704.0, 0.1,
                 kind="mixed", n_inst=(50, 50), radius=(10.0, 120.0)),
}

# bin counts of the sweep on workload 5 (Table 1 of the paper)
SWEEP_BINS = (8, 16, 32, 64, 80)


def rng_for(config: int, *extra: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_BASE, config, *extra])))


@dataclass
class Frame:
    spec: FrameSpec
    emb: np.ndarray            # [H][W][D], spec dtype
    fg: np.ndarray             # [H][W], spec dtype
    inst: np.ndarray           # [H][W] int32, 0 = background
    centroids: np.ndarray      # [N][2] (x, y) fp64 of the kept instances, index = id-1
    kept: np.ndarray           # [N] bool, instance has at least one pixel
    outliers: Optional[np.ndarray] = None
    meta: dict = field(default_factory=dict)

    @property
    def fg_fraction(self) -> float:
        return float((self.inst > 0).mean())


# --------------------------------------------------------------------------
# rasterisation on pixel centres
# --------------------------------------------------------------------------
def _raster_ellipse(inst, k, cx, cy, ra, rb, theta):
    H, W = inst.shape
    R = max(ra, rb)
    x0, x1 = max(0, int(math.floor(cx - R - 1))), min(W, int(math.ceil(cx + R + 1)))
    y0, y1 = max(0, int(math.floor(cy - R - 1))), min(H, int(math.ceil(cy + R + 1)))
    if x0 >= x1 or y0 >= y1:
        return
    xs = np.arange(x0, x1) + 0.5 - cx
    ys = np.arange(y0, y1) + 0.5 - cy
    dx, dy = np.meshgrid(xs, ys)
    c, s = math.cos(theta), math.sin(theta)
    u = (dx * c + dy * s) / ra
    v = (-dx * s + dy * c) / rb
    m = (u * u + v * v) <= 1.0
    inst[y0:y1, x0:x1][m] = k


def _raster_polygon(inst, k, cx, cy, r, angles):
    H, W = inst.shape
    vx = cx + r * np.cos(angles)
    vy = cy + r * np.sin(angles)
    x0, x1 = max(0, int(math.floor(vx.min() - 1))), min(W, int(math.ceil(vx.max() + 1)))
    y0, y1 = max(0, int(math.floor(vy.min() - 1))), min(H, int(math.ceil(vy.max() + 1)))
    if x0 >= x1 or y0 >= y1:
        return
    px, py = np.meshgrid(np.arange(x0, x1) + 0.5, np.arange(y0, y1) + 0.5)
    m = np.ones(px.shape, dtype=bool)
    n = len(angles)
    for i in range(n):
        ax, ay = vx[i], vy[i]
        bx, by = vx[(i + 1) % n], vy[(i + 1) % n]
        m &= ((bx - ax) * (py - ay) - (by - ay) * (px - ax)) >= 0.0
    inst[y0:y1, x0:x1][m] = k


def _draw_instances(spec: FrameSpec, rng: np.random.Generator, n: int, H: int, W: int):
    inst = np.zeros((H, W), dtype=np.int32)
    shapes = []
    for k in range(1, n + 1):
        if spec.kind == "mixed":
            kind = "ellipse" if rng.random() < 0.5 else "polygon"
        else:
            kind = spec.kind
        if spec.radius_law == "rowdep":
            cy = H * rng.random() ** 1.5
            cx = W * rng.random()
            r = 4.0 * 50.0 ** math.sqrt(cy / H) * math.exp(rng.normal(0.0, 0.2))
            r = min(max(r, spec.radius[0]), spec.radius[1])
        else:
            cx = W * rng.random()
            cy = H * rng.random()
            lo, hi = spec.radius
            if spec.radius_law == "loguniform":
                r = math.exp(rng.uniform(math.log(lo), math.log(hi)))
            else:  # "uniform" and "semi" both draw the first size uniformly
                r = rng.uniform(lo, hi)
        if kind == "ellipse":
            if spec.radius_law == "semi":
                rb = rng.uniform(*spec.radius)
            else:
                rb = r * rng.uniform(0.5, 1.0)
            theta = rng.uniform(0.0, math.pi)
            _raster_ellipse(inst, k, cx, cy, r, rb, theta)
            shapes.append(("ellipse", cx, cy, r, rb, theta))
        else:
            nv = int(rng.integers(5, 10))
            ang = np.sort(rng.uniform(0.0, 2.0 * math.pi, size=nv))
            _raster_polygon(inst, k, cx, cy, r, ang)
            shapes.append(("polygon", cx, cy, r, ang))
    return inst, shapes


def encode_positions(x, y, fx, fy) -> np.ndarray:
    """Target encoding (Eq1/Eq2 layout) of positions x, y (pixels) -> [..., 4F] fp64."""
    x = np.asarray(x, dtype=np.float64)[..., None]
    y = np.asarray(y, dtype=np.float64)[..., None]
    F = len(fx)
    out = np.empty(x.shape[:-1] + (4 * F,), dtype=np.float64)
    out[..., 0:2 * F:2] = np.sin(x * fx)
    out[..., 1:2 * F:2] = np.cos(x * fx)
    out[..., 2 * F::2] = np.sin(y * fy)
    out[..., 2 * F + 1::2] = np.cos(y * fy)
    return out


def centroids_of(inst: np.ndarray, n: int):
    """fp64 mean of the visible pixel centres of ids 1..n; (cent[n,2], kept[n])."""
    H, W = inst.shape
    ids = inst.ravel()
    cnt = np.bincount(ids, minlength=n + 1)[1:n + 1].astype(np.float64)
    jj = np.tile(np.arange(W, dtype=np.float64) + 0.5, H)
    ii = np.repeat(np.arange(H, dtype=np.float64) + 0.5, W)
    sx = np.bincount(ids, weights=jj, minlength=n + 1)[1:n + 1]
    sy = np.bincount(ids, weights=ii, minlength=n + 1)[1:n + 1]
    kept = cnt > 0
    cent = np.zeros((n, 2), dtype=np.float64)
    cent[kept, 0] = sx[kept] / cnt[kept]
    cent[kept, 1] = sy[kept] / cnt[kept]
    return cent, kept


def make_frame(config: int, frame: int = 0, *, calibration: bool = False, spec: Optional[FrameSpec] = None) -> Frame:
    """Draw frame ``frame`` of workload ``config`` (or of an explicit ``spec``)."""
    spec = spec if spec is not None else CONFIGS[config]
    extra = (999,) if calibration else ((frame,) if spec.n_frames > 1 else ())
    rng = rng_for(config, *extra)
    H, W, F = spec.H, spec.W, spec.n_freq
    lo, hi = spec.n_inst
    n = lo if lo == hi else int(rng.integers(lo, hi + 1))
    inst, shapes = _draw_instances(spec, rng, n, H, W)
    cent, kept = centroids_of(inst, n)
    fx, fy = spec.freqs()

    table = np.zeros((n + 1, 4 * F), dtype=np.float64)
    if n:
        table[1:] = encode_positions(cent[:, 0], cent[:, 1], fx, fy)
    clean = table.astype(np.float32)[inst]                 # [H][W][D]
    outliers = None
    if spec.outlier_frac > 0.0:
        n_out = int(round(spec.outlier_frac * H * W))
        outliers = rng.choice(H * W, size=n_out, replace=False)
        ox = W * rng.random(n_out)
        oy = H * rng.random(n_out)
        clean.reshape(H * W, 4 * F)[outliers] = encode_positions(ox, oy, fx, fy).astype(np.float32)
    noise = rng.standard_normal((H, W, 4 * F), dtype=np.float32)
    noise *= np.float32(spec.sigma)
    clean += noise
    del noise
    emb = clean.astype(spec.np_dtype)
    del clean
    fgn = rng.standard_normal((H, W), dtype=np.float32) * np.float32(spec.fg_sigma)
    fg = ((inst > 0).astype(np.float32) + fgn).astype(spec.np_dtype)
    return Frame(spec, emb, fg, inst, cent, kept, outliers, {"n_drawn": n, "shapes": shapes})
