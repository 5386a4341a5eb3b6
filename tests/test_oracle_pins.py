"""Pins of the CPU oracle against facts fixed by the paper and the mathematics.

None of these re-types the oracle's loops: the checks are closed forms, the
paper's matrix form of the vote (Eq11) evaluated in fp64 by numpy within a
derived error bound, a library local-maximum filter, a pure-Python exhaustive
search on tiny frames, a noise-free special case whose answer is known in
advance, and invariants of the decoder's definition.
"""
import math

import numpy as np
import pytest

import oracle
from paper_2609_16874_amd import synth
from tests import refmath


def paper_freqs(H, W, L=4):
    """The paper's L harmonics (Eq2) in rad/px: 2^l pi over the normalised axis."""
    fx = np.array([2.0 * math.pi * 2 ** l / W for l in range(L)])
    fy = np.array([2.0 * math.pi * 2 ** l / H for l in range(L)])
    return fx, fy


# --------------------------------------------------------------------------
# S0 constants
# --------------------------------------------------------------------------
def _tiny_decode(bins_w=32, bins_h=32, H=8, W=8, F=4):
    emb = np.zeros((H, W, 4 * F), np.float32)
    fg = np.zeros((H, W), np.float32)
    fx, fy = paper_freqs(H, W, F)
    return oracle.decode(emb, fg, fx, fy, bins_w, bins_h, 4, 0.5, 0.0), fx, fy


def test_weight_buckets_bound_e_minus_d_over_each_bucket():
    """Every weight bucket's entry lies between 2^15 e^-d at the bucket's
    largest and smallest squared distance (d = sqrt(S)/4096: the Euclidean
    distance of Eq4 in embedding units); S = 0 weighs exactly 2^15."""
    res = _tiny_decode()[0]
    wt = res["weights"].astype(np.int64)
    assert len(wt) == 8192 and wt[0] == 32768
    checked = 0
    for key in range(8192):
        r = refmath.bucket_range(key, 8)
        if r is None:
            continue
        d_lo, d_hi = math.sqrt(r[0]) / 4096, math.sqrt(r[1]) / 4096
        assert round(32768 * math.exp(-d_hi)) - 1 <= wt[key] <= round(32768 * math.exp(-d_lo)) + 1, key
        checked += 1
    assert checked > 4000
    # beyond the binades too small to hold several integers the weights fall
    # with the distance
    assert np.all(np.diff(wt[256 * 12:]) <= 0)


def test_distance_of_exact_offsets_from_a_palette_entry():
    """Eq4 in closed form: a pixel whose x block is the palette entry of bin
    a0 moved by (3, 4) units of 1/4096 on two channels, and whose y block is
    the entry of b0 moved by k units on one channel, is at distance exactly
    5 + k units (both squared distances are perfect squares, whose binary32
    roots are exact), so its score is e^-((5 + k)/4096); k = 0 on both axes
    gives the score 1 exactly."""
    H, W, F, bins = 8, 8, 2, 3
    res, fx, fy = _tiny_decode(bins_w=bins, bins_h=bins, H=H, W=W, F=F)
    a0, b0 = 1, 1
    px = res["pal_x"][a0].astype(np.float64)
    py = res["pal_y"][b0].astype(np.float64)
    emb = np.zeros((H, W, 4 * F), np.float32)
    k = np.arange(H * W).reshape(H, W) % 7
    emb[..., :2 * F] = px / 4096.0
    emb[..., 2 * F:] = py / 4096.0
    xy = np.arange(H * W).reshape(H, W) % 2 == 1
    emb[xy, 0] += 3.0 / 4096.0
    emb[xy, 1] += 4.0 / 4096.0
    emb[..., 2 * F + 1] += k / 4096.0
    fg = np.ones((H, W), np.float32)
    r = oracle.decode(emb, fg, fx, fy, bins, bins, 4, 0.5, 0.0)
    assert r["K"] == 1 and (r["centroids"]["bin_x"][0], r["centroids"]["bin_y"][0]) == (a0, b0)
    assert np.all(r["labels"] == 1)
    d = np.where(xy, 5, 0) + k
    np.testing.assert_allclose(r["score_map"], np.exp(-d / 4096.0), rtol=2e-7, atol=0)
    assert r["score_map"][0, 0] == 1.0


def test_palette_is_gamma_at_bin_centres():
    """Eq9: each palette row is 4096*gamma(bin centre) rounded (|err| <= 1/2),
    with the x block / y block and (sin, cos) layout of Eq1/Eq3."""
    H, W = 48, 80
    res, fx, fy = _tiny_decode(bins_w=7, bins_h=5, H=H, W=W)
    px, py = refmath.palettes_real(H, W, fx, fy, 7, 5)
    assert np.abs(res["pal_x"] - 4096.0 * px).max() <= 0.5 + 1e-9
    assert np.abs(res["pal_y"] - 4096.0 * py).max() <= 0.5 + 1e-9


def test_palette_unit_circle_and_mirror():
    """sin^2 + cos^2 = 1 per harmonic; mirror symmetry about the frame centre
    when every harmonic completes whole periods over the axis."""
    H = W = 64
    res, fx, fy = _tiny_decode(bins_w=32, bins_h=32, H=H, W=W, F=8)
    P = res["pal_x"].astype(np.int64)
    F = 8
    pair = P[:, 0::2] ** 2 + P[:, 1::2] ** 2
    assert np.abs(pair - 4096 ** 2).max() <= 4096 * math.sqrt(2) + 0.5
    assert np.abs(P[::-1, 0::2] + P[:, 0::2]).max() <= 1
    assert np.abs(P[::-1, 1::2] - P[:, 1::2]).max() <= 1
    assert P.shape == (32, 2 * F)


# --------------------------------------------------------------------------
# S1+S2: the vote histogram against the paper's matrix form
# --------------------------------------------------------------------------
@pytest.mark.parametrize("dtype,F,bins", [(np.float32, 4, 12), (np.float16, 4, 9), (np.float32, 8, 16),
                                          (np.float16, 16, 32)])
def test_histogram_matches_eq11_within_quantisation_bound(dtype, F, bins):
    rng = np.random.default_rng(11 + F + bins)
    H, W = 24, 31
    fx, fy = paper_freqs(H, W, F)
    # a few instances with random centroids, small noise (no clamping)
    inst = rng.integers(0, 4, size=(H, W))
    cx, cy = rng.uniform(0, W, 4), rng.uniform(0, H, 4)
    clean = synth.encode_positions(cx[inst], cy[inst], fx, fy)
    emb = (clean + 0.05 * rng.standard_normal(clean.shape)).astype(dtype)
    fg = (inst > 0).astype(dtype)
    assert np.abs(emb.astype(np.float64)).max() < 1.5
    res = oracle.decode(emb, fg, fx, fy, bins, bins, 8, 0.5, 0.0)
    h_real, ex, ey = refmath.real_histogram(emb, fg, fx, fy, bins, bins)
    h_can = res["hist"].astype(np.float64) * 2.0 ** -30
    bound = refmath.quant_bound(ex, ey, 2 * F)
    assert np.all(np.abs(h_can - h_real) <= bound)
    # the bound is tight enough to catch a transposed histogram
    assert not np.all(np.abs(h_can.T - h_real.T[::-1]) <= bound)


def test_histogram_catches_axis_swap():
    """A decoder that swapped the x and y blocks would miss the bound."""
    rng = np.random.default_rng(5)
    H, W, F = 20, 20, 4
    fx, fy = paper_freqs(H, W, F)
    inst = rng.integers(0, 3, size=(H, W))
    cx, cy = np.array([0, 3.0, 15.0]), np.array([0, 17.0, 4.0])
    emb = synth.encode_positions(cx[inst], cy[inst], fx, fy).astype(np.float32)
    fg = (inst > 0).astype(np.float32)
    res = oracle.decode(emb, fg, fx, fy, 10, 10, 8, 0.5, 0.0)
    swapped = np.concatenate([emb[..., 2 * F:], emb[..., :2 * F]], -1)
    h_real, ex, ey = refmath.real_histogram(swapped, fg, fx, fy, 10, 10)
    bound = refmath.quant_bound(ex, ey, 2 * F)
    assert not np.all(np.abs(res["hist"] * 2.0 ** -30 - h_real) <= bound)


# --------------------------------------------------------------------------
# S3: local maxima against a library filter
# --------------------------------------------------------------------------
@pytest.mark.parametrize("cfg", [0, 1])
def test_peaks_match_library_local_max(cfg):
    f = synth.make_frame(cfg)
    res = oracle.decode_frame(f, peak_threshold=0.3, capacity=1024)
    cut = math.floor(0.3 * 2 ** 30)
    m = refmath.strict_local_maxima(res["hist"].astype(np.int64), cut)
    bb, aa = np.nonzero(m)                      # row-major = ascending b*Bw + a
    assert res["K"] == len(aa)
    assert np.array_equal(res["centroids"]["bin_x"], aa)
    assert np.array_equal(res["centroids"]["bin_y"], bb)
    assert np.all(res["centroids"]["score"] > 0.3)


def test_plateau_gives_no_peak_and_single_bin_is_a_peak():
    H = W = 6
    F = 2
    fx, fy = paper_freqs(H, W, F)
    emb = np.zeros((H, W, 4 * F), np.float32)
    fg = np.zeros((H, W), np.float32)          # empty S: H == 0 everywhere
    r = oracle.decode(emb, fg, fx, fy, 5, 5, 4, 0.5, -1.0)
    assert r["K"] == 0 and not r["labels"].any()
    r1 = oracle.decode(emb, fg, fx, fy, 1, 1, 4, 0.5, -1.0)
    assert r1["K"] == 1 and not r1["labels"].any()


# --------------------------------------------------------------------------
# whole decoder: pure-Python exhaustive search on tiny frames
# --------------------------------------------------------------------------
@pytest.mark.parametrize("seed,dtype,F,bw,bh,cap", [(0, np.float32, 2, 5, 4, 6), (1, np.float16, 3, 6, 6, 2),
                                                    (2, np.float32, 1, 3, 7, 8), (3, np.float16, 4, 8, 5, 1)])
def test_oracle_equals_exhaustive_search(seed, dtype, F, bw, bh, cap):
    rng = np.random.default_rng(seed)
    H, W = 7, 9
    fx, fy = paper_freqs(H, W, F)
    inst = rng.integers(0, 4, size=(H, W))
    cx, cy = rng.uniform(0, W, 4), rng.uniform(0, H, 4)
    emb = (synth.encode_positions(cx[inst], cy[inst], fx, fy) + 0.2 * rng.standard_normal((H, W, 4 * F))).astype(dtype)
    fg = ((inst > 0) + 0.05 * rng.standard_normal((H, W))).astype(dtype)
    theta = 0.05 * (inst > 0).sum()
    dist = {}
    hist, peaks, K, labels = refmath.brute_decode(emb, fg, fx, fy, bw, bh, cap, 0.5, theta, dist_out=dist)
    res = oracle.decode(emb, fg, fx, fy, bw, bh, cap, 0.5, theta)
    assert np.array_equal(res["hist"], np.array(hist, dtype=np.uint64))
    assert res["K"] == K
    got = list(zip(res["centroids"]["bin_x"].tolist(), res["centroids"]["bin_y"].tolist()))
    assert got == peaks[:cap]
    assert np.array_equal(res["labels"], np.array(labels, dtype=np.int32))
    # the score map is e^-(winning distance sum / 4096)
    assert dist or K == 0
    for (i, j), d in dist.items():
        assert abs(float(res["score_map"][i, j]) - math.exp(-d / 4096.0)) <= 1e-6 * math.exp(-d / 4096.0)


# --------------------------------------------------------------------------
# Eq8 mask threshold and the all-pixels participation of Section 3.1
# --------------------------------------------------------------------------
def _tiny_frame(seed, dtype, F, H=7, W=9):
    rng = np.random.default_rng(seed)
    fx, fy = paper_freqs(H, W, F)
    inst = rng.integers(0, 4, size=(H, W))
    cx, cy = rng.uniform(0, W, 4), rng.uniform(0, H, 4)
    emb = (synth.encode_positions(cx[inst], cy[inst], fx, fy) + 0.2 * rng.standard_normal((H, W, 4 * F))).astype(dtype)
    fg = ((inst > 0) + 0.05 * rng.standard_normal((H, W))).astype(dtype)
    return emb, fg, inst, fx, fy


# tau = (q, off): the winning code sum at quantile q of the pixels, plus off,
# over 4096; off = 0 puts pixels exactly on the threshold, where the strict
# test of Eq8 decides
@pytest.mark.parametrize("seed,dtype,F,bw,bh,cap,use_fg,tau", [
    (4, np.float32, 2, 5, 4, 6, True, (0.3, 0.5)), (5, np.float16, 3, 6, 6, 3, False, (0.7, 0.5)),
    (6, np.float32, 1, 4, 7, 8, False, (0.5, 0)), (7, np.float32, 2, 6, 5, 4, True, (0.4, 0)),
    (8, np.float16, 2, 5, 5, 4, True, 0.0)])
def test_mask_threshold_and_all_pixels_equal_exhaustive_search(seed, dtype, F, bw, bh, cap, use_fg, tau):
    emb, fg, inst, fx, fy = _tiny_frame(seed, dtype, F)
    fg = fg if use_fg else None
    theta = 0.05 * (inst > 0).sum()
    if isinstance(tau, tuple):
        d = {}
        refmath.brute_decode(emb, fg, fx, fy, bw, bh, cap, 0.5, theta, dist_out=d)
        vals = sorted(d.values())
        tau = (vals[int(tau[0] * len(vals))] + tau[1]) / 4096.0
    hist, peaks, K, labels = refmath.brute_decode(emb, fg, fx, fy, bw, bh, cap, 0.5, theta, tau)
    res = oracle.decode(emb, fg, fx, fy, bw, bh, cap, 0.5, theta, tau=tau)
    assert np.array_equal(res["hist"], np.array(hist, dtype=np.uint64))
    assert res["K"] == K
    lab = np.array(labels, dtype=np.int32)
    assert np.array_equal(res["labels"], lab)
    assert np.array_equal(res["centroids"]["npix"], np.bincount(lab.ravel(), minlength=min(K, cap) + 1)[1:])


def test_mask_threshold_on_noise_free_frame_with_all_pixels():
    """Every pixel votes (no fg channel).  Instance pixels sit within
    snap_distance(F) of their own bin; background pixels carry a zero
    embedding, at distance sqrt(F) per axis from every bin (|gamma|^2 = F),
    so each adds about e^(-2 sqrt F) to every bin: a threshold above that
    level plus half the smallest instance finds exactly the instances.  A
    tau just above twice the snap distance then keeps exactly the instance
    pixels, and tau = 0 keeps nothing (Eq8 is strict)."""
    H = W = 96
    bins, F = 16, 4
    cells = [(3, 3), (11, 4), (3, 12), (12, 12), (8, 8)]
    emb, fg, inst, fx, fy = _snapped_frame(H, W, bins, cells, half=5, F=F)
    sizes = np.bincount(inst.ravel())
    floor = sizes[0] * math.exp(-2.0 * math.sqrt(F)) * 1.02
    theta = floor + 0.5 * sizes[1:].min()
    want = sorted(cells, key=lambda ab: ab[1] * bins + ab[0])
    rank = {ab: i + 1 for i, ab in enumerate(want)}
    expect = np.zeros_like(inst)
    for k, ab in enumerate(cells, start=1):
        expect[inst == k] = rank[ab]
    tau = 2.0 * snap_distance(F) * (1 + 2.0 ** -20)              # sqrt rounding: 2^-24 relative per axis
    assert tau < math.sqrt(F)
    res = oracle.decode(emb, None, fx, fy, bins, bins, 64, 0.5, theta, tau=tau)
    got = list(zip(res["centroids"]["bin_x"].tolist(), res["centroids"]["bin_y"].tolist()))
    assert res["K"] == len(cells) and got == want
    assert np.array_equal(res["labels"], expect)
    assert np.array_equal(res["centroids"]["npix"], np.bincount(expect.ravel(), minlength=len(cells) + 1)[1:])
    assert np.all(res["score_map"][expect > 0] >= np.float32(math.exp(-tau)))
    assert not res["score_map"][expect == 0].any()
    # no threshold: every pixel is labelled, the instances as before
    full = oracle.decode(emb, None, fx, fy, bins, bins, 64, 0.5, theta)
    assert np.all(full["labels"] > 0) and np.array_equal(full["labels"][expect > 0], expect[expect > 0])
    assert full["centroids"]["npix"].sum() == H * W
    zero = oracle.decode(emb, None, fx, fy, bins, bins, 64, 0.5, theta, tau=0.0)
    assert zero["K"] == len(cells) and not zero["labels"].any() and not zero["centroids"]["npix"].any()


def test_mask_threshold_nests():
    """Raising tau only adds pixels, each with its tau = inf label; the
    histogram and the centroids do not depend on tau; counts follow labels;
    and the kept pixels are those whose affinity e^-d (the paper's kernel
    compares affinities with e^-tau) exceeds e^-tau, where d is read back
    from the tau = inf score map."""
    f = synth.make_frame(0)
    base = oracle.decode_frame(f, peak_threshold=0.5)
    lab0 = base["labels"]
    d = np.full(lab0.shape, np.inf)
    d[lab0 > 0] = -np.log(base["score_map"][lab0 > 0].astype(np.float64))
    prev = np.zeros(lab0.shape, dtype=bool)
    for tau in (0.0, 0.25, 0.5, 1.0, 2.0, 8.0):
        r = oracle.decode_frame(f, peak_threshold=0.5, tau=tau)
        assert np.array_equal(r["hist"], base["hist"]) and r["K"] == base["K"]
        keep = r["labels"] > 0
        assert np.all(prev <= keep) and np.all(keep <= (lab0 > 0))
        assert np.array_equal(r["labels"][keep], lab0[keep])
        assert np.array_equal(r["centroids"]["npix"],
                              np.bincount(r["labels"].ravel(), minlength=len(r["centroids"]) + 1)[1:])
        # away from the boundary (float rounding of expf) the sets agree
        clear = np.abs(d - tau) > 1e-5
        assert np.array_equal(keep[clear], (d < tau)[clear])
        prev = keep
    assert 0 < prev.sum() and prev.sum() <= (lab0 > 0).sum()


# --------------------------------------------------------------------------
# noise-free special case: exact recovery of the generating centroids
# --------------------------------------------------------------------------
def snap_distance(F):
    """Largest canonical distance between the fp32 encoding of a bin centre
    and that bin's palette entry: both are 4096 gamma rounded to an integer,
    of values within 4096 * 2^-25 of each other (the fp32 cast), so they
    differ by at most one unit of 1/4096 per channel: sqrt(2F)/4096."""
    return math.sqrt(2 * F) / 4096


def _snapped_frame(H, W, bins, cells, half, F=4):
    """Square instances centred on chosen bin centres; the embedding is the
    encoding of that exact bin centre, so every instance pixel is within
    snap_distance(F) of its own bin."""
    fx, fy = paper_freqs(H, W, F)
    xa = refmath.bin_centres(bins, W)
    yb = refmath.bin_centres(bins, H)
    inst = np.zeros((H, W), np.int32)
    for k, (a, b) in enumerate(cells, start=1):
        x0, y0 = int(xa[a]), int(yb[b])
        inst[max(0, y0 - half):y0 + half, max(0, x0 - half):x0 + half] = k
    cx = np.concatenate([[0.0], [xa[a] for a, _ in cells]])
    cy = np.concatenate([[0.0], [yb[b] for _, b in cells]])
    emb = synth.encode_positions(cx[inst], cy[inst], fx, fy)
    emb[inst == 0] = 0.0
    return emb.astype(np.float32), (inst > 0).astype(np.float32), inst, fx, fy


@pytest.mark.parametrize("order", [0, 1])
def test_noise_free_decodes_generating_centroids_and_labels(order):
    H = W = 96
    bins = 16
    # two instances share a column and two share a row, so an assignment that
    # ignored one axis would tie and mislabel them
    cells = [(3, 3), (11, 4), (3, 12), (12, 12), (8, 8)]
    if order:
        cells = cells[::-1]                     # instance order must not matter
    emb, fg, inst, fx, fy = _snapped_frame(H, W, bins, cells, half=5)
    sizes = np.bincount(inst.ravel())[1:]
    theta = 0.5 * sizes.min()
    res = oracle.decode(emb, fg, fx, fy, bins, bins, 64, 0.5, theta)
    got = sorted(zip(res["centroids"]["bin_x"].tolist(), res["centroids"]["bin_y"].tolist()),
                 key=lambda ab: ab[1] * bins + ab[0])
    want = sorted(cells, key=lambda ab: ab[1] * bins + ab[0])
    assert res["K"] == len(cells) and got == want
    # labels equal the generating map up to the bin-order renumbering
    rank = {ab: i + 1 for i, ab in enumerate(want)}
    expect = np.zeros_like(inst)
    for k, ab in enumerate(cells, start=1):
        expect[inst == k] = rank[ab]
    assert np.array_equal(res["labels"], expect)
    assert np.array_equal(res["centroids"]["npix"], np.bincount(expect.ravel(), minlength=len(cells) + 1)[1:])
    # a distance of at most snap_distance per axis weighs at least
    # e^-snap_distance (up to the table's rounding): score >= |Omega_k| e^-2d
    w = math.exp(-2.0 * snap_distance(4) * (1 + 2.0 ** -8)) - 2.0 ** -14
    for c in res["centroids"]:
        k = [kk for kk, ab in enumerate(cells, start=1) if ab == (c["bin_x"], c["bin_y"])][0]
        assert c["score"] >= sizes[k - 1] * w


# --------------------------------------------------------------------------
# invariants on the workloads
# --------------------------------------------------------------------------
@pytest.mark.parametrize("cfg", [0, 1])
def test_invariants(cfg):
    f = synth.make_frame(cfg)
    theta = 0.5
    res = oracle.decode_frame(f, peak_threshold=theta)
    lab = res["labels"]
    cents = res["centroids"]
    K = res["K"]
    bins = f.spec.bins
    S = f.fg.astype(np.float32) > np.float32(f.spec.fg_threshold)
    assert 1 <= K <= ((bins + 1) // 2) ** 2
    assert np.array_equal(lab > 0, S)                       # partition of the foreground
    assert lab.max() <= len(cents)
    assert cents["npix"].sum() == S.sum()
    assert np.array_equal(cents["npix"], np.bincount(lab.ravel(), minlength=len(cents) + 1)[1:])
    idx = cents["bin_y"] * bins + cents["bin_x"]
    assert np.all(np.diff(idx) > 0)
    a, b = cents["bin_x"], cents["bin_y"]
    cheb = np.maximum(np.abs(a[:, None] - a[None]), np.abs(b[:, None] - b[None]))
    np.fill_diagonal(cheb, 99)
    assert cheb.min() >= 2
    assert np.all(cents["score"] > theta)
    xa = refmath.bin_centres(bins, f.spec.W).astype(np.float32)
    assert np.array_equal(cents["x"], xa[a])


def test_pixel_permutation_invariance():
    """H is a sum over S and each label depends only on its own pixel, so
    permuting the pixels of a frame permutes the labels and nothing else."""
    f = synth.make_frame(0)
    rng = np.random.default_rng(3)
    H, W, D = f.emb.shape
    perm = rng.permutation(H * W)
    emb2 = f.emb.reshape(-1, D)[perm].reshape(H, W, D)
    fg2 = f.fg.reshape(-1)[perm].reshape(H, W)
    fx, fy = f.spec.freqs()
    r1 = oracle.decode(f.emb, f.fg, fx, fy, 32, 32, None, 0.5, 0.5)
    r2 = oracle.decode(emb2, fg2, fx, fy, 32, 32, None, 0.5, 0.5)
    assert np.array_equal(r1["hist"], r2["hist"])
    assert np.array_equal(r1["centroids"], r2["centroids"])
    assert np.array_equal(r1["labels"].reshape(-1)[perm], r2["labels"].reshape(-1))


def test_capacity_overflow_and_empty():
    f = synth.make_frame(0)
    full = oracle.decode_frame(f, peak_threshold=0.5)
    small = oracle.decode_frame(f, peak_threshold=0.5, capacity=3)
    assert small["K"] == full["K"] and len(small["centroids"]) == 3
    assert np.array_equal(small["centroids"][["bin_x", "bin_y", "score"]], full["centroids"][:3][["bin_x", "bin_y", "score"]])
    assert small["labels"].max() == 3
    none = oracle.decode_frame(f, peak_threshold=1e9)
    assert none["K"] == 0 and not none["labels"].any() and not none["score_map"].any()


def test_score_map_is_exp_of_distance():
    f = synth.make_frame(0)
    res = oracle.decode_frame(f, peak_threshold=0.5)
    lab = res["labels"]
    sm = res["score_map"]
    assert np.all(sm[lab == 0] == 0)
    assert np.all((sm[lab > 0] > 0) & (sm[lab > 0] <= 1))


def test_real_mode_close_to_canonical():
    """Diagnostic: the canonical arithmetic changes very few decisions."""
    f = synth.make_frame(1)
    fx, fy = f.spec.freqs()
    can = oracle.decode_frame(f, peak_threshold=2.0)
    real = oracle.decode_real(f.emb, f.fg, fx, fy, 32, 32, None, 0.5, 2.0)
    assert real["K"] == can["K"]
    fgm = f.fg.astype(np.float32) > 0.5
    assert (real["labels"][fgm] == can["labels"][fgm]).mean() > 0.995


def test_argument_errors():
    emb = np.zeros((4, 4, 16), np.float32)
    fg = np.zeros((4, 4), np.float32)
    fx, fy = paper_freqs(4, 4, 4)
    for kw in [dict(bins_w=0), dict(bins_h=129), dict(capacity=0), dict(fg_threshold=float("nan")),
               dict(peak_threshold=float("nan"))]:
        args = dict(bins_w=4, bins_h=4, capacity=4, fg_threshold=0.5, peak_threshold=0.0)
        args.update(kw)
        assert oracle.decode(emb, fg, fx, fy, check=False, **args)["rc"] == 1
    assert oracle.decode(emb[..., :12], fg, fx, fy, 4, 4, 4, 0.5, 0.0, check=False)["rc"] == 1
    # more channels than 4 n_freq are allowed (low harmonics only), an odd count is not
    assert oracle.decode(np.zeros((4, 4, 18), np.float32), fg, fx, fy, 4, 4, 4, 0.5, 0.0, check=False)["rc"] == 0
    assert oracle.decode(np.zeros((4, 4, 17), np.float32), fg, fx, fy, 4, 4, 4, 0.5, 0.0, check=False)["rc"] == 1


# --------------------------------------------------------------------------
# Low harmonics of a longer encoding (the "resolved harmonics" decode)
# --------------------------------------------------------------------------
def low_harmonic_channels(emb, F_used):
    """The channels of the first F_used harmonics of each axis block of a
    [H][W][D] embedding (x block first, then y, each (sin, cos) pairs of
    ascending harmonics, Eq2/Eq3), as a [H][W][4 F_used] array."""
    half = emb.shape[-1] // 2
    return np.concatenate([emb[..., :2 * F_used], emb[..., half:half + 2 * F_used]], axis=-1)


@pytest.mark.parametrize("cfg,F_used", [(0, 1), (0, 3), (0, 4), (0, 8), (2, 4)])
def test_low_harmonics_equal_decoding_the_sliced_encoding(cfg, F_used):
    """Decoding a D-channel map with its first F' harmonics is, by definition,
    decoding the map cut down to those 4 F' channels (Eq9/Eq10 compare each
    axis block with palettes of the same harmonics)."""
    f = synth.make_frame(cfg)
    if cfg == 2:      # a 128 x 160 window keeps the full-size frame's instances and layout
        emb, fg = f.emb[256:384, 240:400], f.fg[256:384, 240:400]
        H, W = emb.shape[:2]
        fx = np.array([2.0 * math.pi * 2 ** k / 640 for k in range(f.spec.n_freq)])
        fy = fx.copy()
    else:
        emb, fg = f.emb, f.fg
        H, W = emb.shape[:2]
        fx, fy = f.spec.freqs()
    fx, fy = fx[:F_used], fy[:F_used]
    bins = 16
    theta = 0.02 * H * W / 1024
    full = oracle.decode(emb, fg, fx, fy, bins, bins, 64, 0.5, theta)
    cut = oracle.decode(low_harmonic_channels(emb, F_used), fg, fx, fy, bins, bins, 64, 0.5, theta)
    assert full["K"] == cut["K"]
    assert np.array_equal(full["hist"], cut["hist"])
    assert np.array_equal(full["centroids"], cut["centroids"])
    assert np.array_equal(full["labels"], cut["labels"])
    assert full["K"] > 0


def test_clamp_saturates():
    """Input reading: values beyond +-1.5 saturate at +-1.5, +-inf likewise,
    and a NaN channel clamps to -1.5 -- so such frames decode exactly like
    their clipped copies."""
    rng = np.random.default_rng(9)
    H, W, F = 6, 7, 2
    fx, fy = paper_freqs(H, W, F)
    base = rng.uniform(-1.0, 1.0, (H, W, 4 * F)).astype(np.float32)
    fg = np.ones((H, W), np.float32)
    wild = base.copy()
    wild[0, 0, 0], wild[1, 2, 3], wild[2, 2, 5] = 7.5, -np.inf, np.nan
    wild[3, 3, 1] = 1e30
    clipped = base.copy()
    clipped[0, 0, 0], clipped[1, 2, 3], clipped[2, 2, 5], clipped[3, 3, 1] = 1.5, -1.5, -1.5, 1.5
    r1 = oracle.decode(wild, fg, fx, fy, 4, 4, 16, 0.5, 0.0)
    r2 = oracle.decode(clipped, fg, fx, fy, 4, 4, 16, 0.5, 0.0)
    assert np.array_equal(r1["hist"], r2["hist"]) and np.array_equal(r1["labels"], r2["labels"])
    unclipped = base.copy()
    unclipped[0, 0, 0] = 1.4                    # inside the range: no saturation
    r3 = oracle.decode(unclipped, fg, fx, fy, 4, 4, 16, 0.5, 0.0)
    assert not np.array_equal(r3["hist"], r2["hist"])


def test_threshold_is_strict():
    """'exceeds a predefined threshold': a peak whose vote mass equals the
    threshold is dropped, one unit below it is kept."""
    f = synth.make_frame(0)
    base = oracle.decode_frame(f, peak_threshold=0.0, capacity=1024)
    top = base["centroids"][np.argmax(base["centroids"]["score"])]
    s = float(top["score"])                     # exactly H * 2^-30
    at = oracle.decode_frame(f, peak_threshold=s, capacity=1024)
    below = oracle.decode_frame(f, peak_threshold=s - 2.0 ** -30, capacity=1024)
    assert at["K"] == 0 and below["K"] == 1
    assert below["centroids"][0]["bin_x"] == top["bin_x"] and below["centroids"][0]["bin_y"] == top["bin_y"]


def test_exact_tie_goes_to_lowest_index():
    """With one harmonic of period W/2 the first and last of three x bins get
    bit-identical palettes, so both are peaks with identical votes and every
    pixel is at exactly the same distance from both: the lower index wins."""
    H = W = 16
    fx = np.array([4.0 * math.pi / W])
    fy = np.array([4.0 * math.pi / H])
    emb = np.zeros((H, W, 4), np.float32)
    emb[..., 0], emb[..., 1] = 0.0, -1.0         # gamma(x = 4) = gamma(x = 12)
    emb[..., 2], emb[..., 3] = 0.0, 1.0
    fg = np.ones((H, W), np.float32)
    res = oracle.decode(emb, fg, fx, fy, 3, 1, 4, 0.5, 1.0)
    assert res["pal_x"][0].tolist() == res["pal_x"][2].tolist()
    assert res["K"] == 2
    assert res["centroids"]["bin_x"].tolist() == [0, 2]
    assert np.all(res["labels"] == 1)
    assert res["centroids"]["npix"].tolist() == [H * W, 0]


def _frozen_threshold(cfg):
    import json
    import os
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "configs.json")
    return json.load(open(path))["configs"][str(cfg)]["peak_threshold"]


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_assignment_agrees_with_eq7_in_fp64(cfg):
    """Eq7 on the unquantised input in fp64 (numpy, here) with the oracle's
    candidates: at most 0.1 % of the foreground is labelled differently, and
    every difference is a near-tie, i.e. the two smallest fp64 distance sums
    lie within what the 1/4096 rounding of input and palette can move them
    (2 sqrt(2F) 2^-12 per sum, twice that between two sums) or the pixel has
    a clamped channel.  The canonical peaks are those of the fp64 real-valued
    histogram (Eq11) with the same threshold."""
    f = synth.make_frame(cfg)
    theta = _frozen_threshold(cfg)
    fx, fy = f.spec.freqs()
    can = oracle.decode_frame(f, peak_threshold=theta)
    real = oracle.decode_real(f.emb, f.fg, fx, fy, 32, 32, None, 0.5, theta)
    a, b = can["centroids"]["bin_x"], can["centroids"]["bin_y"]
    assert real["peaks"].tolist() == (b * 32 + a).tolist()
    lab, sel, gap = refmath.real_labels(f.emb, f.fg, fx, fy, 32, 32, a, b)
    got = can["labels"].reshape(-1)[sel]
    bad = got != lab
    assert bad.mean() <= 1e-3, bad.mean()
    clamped = (np.abs(f.emb.reshape(-1, f.emb.shape[-1])[sel].astype(np.float32)) > 1.5).any(1)
    near = gap < 4.0 * math.sqrt(2 * len(fx)) * 2.0 ** -12
    assert np.all((near | clamped)[bad])


def test_far_pixels_take_the_exact_argmin():
    """Pixels far from every candidate (channels at the clamp bound, squared
    distances near 2^32, where fl32(S) rounds): the label is the lowest
    candidate index among the smallest exact sums sqrtf(fl32(S_x)) +
    sqrtf(fl32(S_y)) (Eq7 with the lowest-index tie rule), by brute force
    over the oracle's palettes."""
    from tests import farframe
    emb, fg, fx, fy, theta, far = farframe.make()
    ref = oracle.decode(emb, fg, fx, fy, farframe.BINS, farframe.BINS, farframe.CAP, 0.5, theta)
    sums, smax = farframe.candidate_distance_sums(ref, emb, farframe.F)
    assert ref["K"] >= 2 and smax[far].min() >= 2 ** 24     # fl32(S) rounds on these pixels
    want = sums.argmin(1) + 1                                 # first index among equal sums
    lab = ref["labels"].reshape(-1)
    assert np.array_equal(lab, want)
    assert len(set(lab[far].tolist())) >= 3          # several different winners among them
    # and the score is e^-(winning sum / 4096)
    np.testing.assert_allclose(ref["score_map"].reshape(-1)[far],
                               np.exp(-sums[far].min(1) / 4096.0).astype(np.float32), rtol=1e-6)


# --------------------------------------------------------------------------
# the fp64 real-valued mode (the reference of the per-tuple ablation)
# --------------------------------------------------------------------------
def _real_case(case):
    if case == "cfg0":
        f = synth.make_frame(0)
        fx, fy = f.spec.freqs()
        return f.emb, f.fg, fx, fy, 32, 32, 0.5
    seed = int(case[-1])
    rng = np.random.default_rng(seed)
    H, W, F = 11, 13, 2 + seed
    fx, fy = paper_freqs(H, W, F)
    inst = rng.integers(0, 4, size=(H, W))
    cx, cy = rng.uniform(0, W, 4), rng.uniform(0, H, 4)
    emb = synth.encode_positions(cx[inst], cy[inst], fx, fy) + 0.2 * rng.standard_normal((H, W, 4 * F))
    emb = emb.astype(np.float32 if seed % 2 else np.float16)
    fg = ((inst > 0) + 0.05 * rng.standard_normal((H, W))).astype(emb.dtype)
    return emb, fg, fx, fy, 7, 6, None


@pytest.mark.parametrize("case", ["tiny0", "tiny1", "tiny2", "cfg0"])
def test_real_mode_equals_matrix_form_library_maxima_and_argmin(case):
    """cpe_oracle_decode_real against three independent restatements: its
    histogram against E_x^T E_y (Eq11, numpy matmul) to fp64 rounding, its
    peaks against a library ring maximum filter on that histogram, and its
    labels against a numpy argmin of fp64 distance sums over its peaks
    (away from fp64 near-ties)."""
    emb, fg, fx, fy, bw, bh, theta = _real_case(case)
    h_ref, _, _ = refmath.real_histogram(emb, fg, fx, fy, bw, bh)
    if theta is None:
        theta = 0.2 * float(h_ref.max())
    real = oracle.decode_real(emb, fg, fx, fy, bw, bh, None, 0.5, theta)
    np.testing.assert_allclose(real["hist"], h_ref, rtol=1e-12, atol=1e-12)
    m = refmath.strict_local_maxima(h_ref, theta)
    bb, aa = np.nonzero(m)
    assert real["K"] == len(aa) > 0
    assert real["peaks"].tolist() == (bb * bw + aa).tolist()
    lab, sel, gap = refmath.real_labels(emb, fg, fx, fy, bw, bh, aa, bb)
    got = real["labels"].reshape(-1)[sel]
    clear = gap > 1e-9
    assert clear.mean() > 0.95
    assert np.array_equal(got[clear], lab[clear])
    assert not real["labels"].reshape(-1)[~sel].any()
