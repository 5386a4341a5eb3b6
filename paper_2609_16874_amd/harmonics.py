"""Which harmonics of a geometric encoding a bin grid resolves.

Host-side configuration of the resolved-harmonics decode, not part of the
decoding arithmetic.  The palettes sample each harmonic at the bin centres
(Eq9); a harmonic whose period along an axis is shorter than a few bin
spacings aliases there, so the per-axis distance profile of a pixel has
several near-equal minima and the vote histogram grows spurious local maxima.
The paper's encoding stops at L = 4 (the shortest period is an eighth of the
axis, about four bin spacings of its 32-bin grid, Section 4.2).  Decoding only
the leading harmonics whose periods span at least ``min_spacings`` bin
spacings keeps that property for longer encodings.
"""
from __future__ import annotations

import math


def resolved_count(freqs, extent: float, bins: int, min_spacings: float = 4.0) -> int:
    """Number of leading harmonics (angular frequencies in rad/pixel, in
    ascending order) whose period is at least ``min_spacings`` bin spacings
    of a ``bins``-bin grid over an axis of ``extent`` pixels (spacing
    extent / (bins + 1), Eq9).  At least 1."""
    spacing = extent / (bins + 1)
    n = 0
    for w in freqs:
        if 2.0 * math.pi / w >= min_spacings * spacing * (1.0 - 1e-12):
            n += 1
        else:
            break
    return max(n, 1)


def resolved_pair(freq_x, freq_y, W: int, H: int, bins_w: int, bins_h: int) -> int:
    """Harmonics to decode on both axes: the smaller of the two counts."""
    return min(resolved_count(freq_x, W, bins_w), resolved_count(freq_y, H, bins_h))
