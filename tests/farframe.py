"""A frame with foreground pixels far from every candidate centroid.

Two instances (left and right halves of a 40 x 48 frame, 16 harmonics per
axis, fp32) plus 40 pixels whose every channel sits at the clamp bound
+-1.5, pointing away from the candidates' palette entries (half of them with
some channels flipped).  Their squared distances reach far above 2^24, where
rounding S to binary32 loses integer precision; the winner is still the Eq7
argmin (smallest exact sum of the two axis distances, then the lowest
candidate index).
"""
import math

import numpy as np

import oracle
from paper_2609_16874_amd import synth

H, W, F = 40, 48, 16
BINS, CAP = 32, 64


def candidate_distance_sums(ref, emb, nf):
    """[pixels][K] Eq7 distance sums of every candidate in units of 1/4096,
    from the oracle's palettes: input on the 1/4096 grid (clamped to
    +-1.5), S exact, r = the float32 square root of S rounded to float32,
    r_x + r_y summed exactly in float64; and per pixel the largest S."""
    v = np.clip(emb.reshape(-1, 4 * nf).astype(np.float32), -1.5, 1.5)
    X = np.rint(np.float32(4096.0) * v).astype(np.int64)

    def dist(Xa, P):
        S = ((Xa[:, None, :] - P[None].astype(np.int64)) ** 2).sum(-1)
        return np.sqrt(S.astype(np.float32)).astype(np.float64), S.max(1)

    rx, sx = dist(X[:, :2 * nf], ref["pal_x"])
    ry, sy = dist(X[:, 2 * nf:], ref["pal_y"])
    A, B = ref["centroids"]["bin_x"], ref["centroids"]["bin_y"]
    return rx[:, A] + ry[:, B], np.maximum(sx, sy)


def make():
    """(emb, fg, fx, fy, theta, far pixel indices)."""
    rng = np.random.default_rng(11)
    fx = np.array([2 * math.pi * 2 ** k / W for k in range(F)]) / 2 ** (F // 2)
    fy = np.array([2 * math.pi * 2 ** k / H for k in range(F)]) / 2 ** (F // 2)
    inst = np.where(np.arange(W)[None, :] < W // 2, 0, 1) * np.ones((H, 1), dtype=int)
    cx0, cy0 = np.array([10.5, 35.2]), np.array([12.3, 27.8])
    emb = synth.encode_positions(cx0[inst], cy0[inst], fx, fy) + 0.02 * rng.standard_normal((H, W, 4 * F))
    emb = emb.astype(np.float32)
    fg = np.ones((H, W), np.float32)
    ref0 = oracle.decode(emb, fg, fx, fy, BINS, BINS, CAP, 0.5, 0.0)
    theta = 0.2 * ref0["hist"].max() * 2.0 ** -30
    ref = oracle.decode(emb, fg, fx, fy, BINS, BINS, CAP, 0.5, theta)
    A, B = ref["centroids"]["bin_x"], ref["centroids"]["bin_y"]
    sx = -np.sign(ref["pal_x"][A].astype(np.float64).sum(0) + 0.5)
    sy = -np.sign(ref["pal_y"][B].astype(np.float64).sum(0) + 0.5)
    far = rng.choice(H * W, 40, replace=False)
    flat = emb.reshape(-1, 4 * F)
    flat[far, :2 * F] = 1.5 * sx
    flat[far, 2 * F:] = 1.5 * sy
    for p in far[20:]:
        flip = rng.random(4 * F) < 0.15
        flat[p, flip] = -flat[p, flip]
    return emb, fg, fx, fy, theta, far
