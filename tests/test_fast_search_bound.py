"""The error bound behind the fast assignment search, on the CPU.

The fast search forms, per batch of one row, the binary32 sum
s = fl32(min over the batch's columns of x~ + y~), where every x~, y~ is a
square root within one binary32 step of the correctly rounded distance
r = sqrt_cr(fl32(S)) (Eq4 on integer squared distances S).  It accepts the
batch with the smallest s when the second smallest exceeds it by at least
8 binary32 steps, which must imply that the exact binary64 minimum D of
that batch is strictly the smallest (Eq7, §3.2 "Mask Aggregation").  These
tests draw near-tied pairs of batches on purpose, perturb every root by one
step either way and check the implication; they also show that a gap of
one step does not suffice, so the threshold is not vacuous.  The threshold
is read from the kernel source; nothing here runs the kernels: numpy's
binary32 square root is correctly rounded.
"""
import os
import re

import numpy as np

_SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                    "paper_2609_16874_amd", "csrc", "k_mfma.hpp")


def _kernel_gap():
    """The threshold the kernel uses (its constexpr kFastGap)."""
    with open(_SRC) as fh:
        m = re.search(r"constexpr int kFastGap = (\d+);", fh.read())
    assert m, "kFastGap not found in k_mfma.hpp"
    return int(m.group(1))


GAP = _kernel_gap()


def _cr(S):
    return np.sqrt(S.astype(np.float32))


def _perturb(r, rng):
    k = rng.integers(-1, 2, size=r.shape)
    up = np.nextafter(r, np.float32(np.inf))
    dn = np.nextafter(r, np.float32(0))
    dn = np.where(r > 0, dn, r)            # the square root of 0 is exact
    return np.where(k > 0, up, np.where(k < 0, dn, r)).astype(np.float32)


def _batches(rng, n, ncol, spread=12):
    """n pairs of batches (w, b) of ncol columns and one row each whose exact
    minima D lie about k binary32 steps apart, k uniform in -spread .. spread."""
    Sxw = rng.integers(0, 2 ** 32, size=(n, ncol), dtype=np.uint64)
    Syw = rng.integers(0, 2 ** 32, size=n, dtype=np.uint64)
    rxw, ryw = _cr(Sxw), _cr(Syw)
    Dw = rxw.astype(np.float64).min(axis=1) + ryw.astype(np.float64)
    # batch b: random columns, and a row chosen so that its sum lands on Dw
    Sxb = rng.integers(0, 2 ** 32, size=(n, ncol), dtype=np.uint64)
    rxb = _cr(Sxb)
    mb = rxb.astype(np.float64).min(axis=1)
    step = np.spacing(Dw.astype(np.float32)).astype(np.float64)
    t = np.clip(Dw + rng.integers(-spread, spread + 1, size=n) * step - mb, 0, 65535.0)
    Syb = np.clip(np.rint(t * t), 0, 2 ** 32 - 1).astype(np.uint64)
    ryb = _cr(Syb)
    Db = mb + ryb.astype(np.float64)
    return (rxw, ryw, Dw), (rxb, ryb, Db)


def _fast_sum(rx, ry, rng):
    xt, yt = _perturb(rx, rng), _perturb(ry, rng)
    m = xt.view(np.uint32).min(axis=1).view(np.float32)     # bit order = value order for r >= 0
    return (m + yt).astype(np.float32)                       # one binary32 rounding


def _steps(a, b):
    return b.view(np.uint32).astype(np.int64) - a.view(np.uint32).astype(np.int64)


def test_the_kernel_threshold_keeps_the_exact_order():
    assert GAP >= 7                 # the error bound's own requirement
    rng = np.random.default_rng(2609)
    checked = 0
    for ncol in (1, 4):
        for _ in range(20):
            (rxw, ryw, Dw), (rxb, ryb, Db) = _batches(rng, 200_000, ncol)
            sw, sb = _fast_sum(rxw, ryw, rng), _fast_sum(rxb, ryb, rng)
            g = _steps(sw, sb)                     # sb above sw by g steps
            acc = g >= GAP
            assert np.all(Db[acc] > Dw[acc])
            acc = -g >= GAP                        # the other way round
            assert np.all(Dw[acc] > Db[acc])
            checked += int(np.count_nonzero((np.abs(g) >= GAP) & (np.abs(g) <= GAP + 2)))
    assert checked > 100_000        # pairs just past the threshold


def test_near_ties_are_drawn_and_one_step_is_not_enough():
    """The draws reach the decision boundary: many pairs fall within the
    threshold, and among them some whose binary32 order (one step apart)
    contradicts the exact order."""
    rng = np.random.default_rng(16874)
    (rxw, ryw, Dw), (rxb, ryb, Db) = _batches(rng, 400_000, 4, spread=2)
    sw, sb = _fast_sum(rxw, ryw, rng), _fast_sum(rxb, ryb, rng)
    g = _steps(sw, sb)
    assert np.count_nonzero(np.abs(g) < GAP) > 10_000
    wrong = ((g >= 1) & (Db <= Dw)) | ((g <= -1) & (Dw <= Db))
    assert np.count_nonzero(wrong) > 0
