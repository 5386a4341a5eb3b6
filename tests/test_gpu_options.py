"""GPU parity of the decode options and of the mask expansion, through the C
ABI, against the CPU oracle.

* cpe_decode_ex with the Eq8 mask threshold tau: thresholds taken from the
  oracle's own distance distribution (the winning distance sums of its tau =
  inf labels, recomputed exactly from its palettes), both on an attained sum
  (the strict test decides pixels sitting exactly on it) and half a unit of
  1/4096 above; tau = 0 and tau = inf.
* cpe_decode_ex without a foreground channel: every pixel votes and is
  labelled (the participating set of Section 3.1), on the matrix-core and the
  generic kernels.
* cpe_decode_masks: the binary masks of Eq8 equal labels == k + 1 byte for
  byte, for aligned and ragged frame sizes, sub-ranges and indices past K.
Bit-exact on histogram, centroids, counts and labels; the score map within
1e-5 relative, as in the main parity suite.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
from paper_2609_16874_amd import synth
from tests.test_gpu_parity import _random_frame, assert_parity, gpu_decode, native, thresholds

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "configs.json")


def code_sums(ref, emb, F):
    """Winning distance sums D (units of 1/4096) of the labelled pixels of an
    oracle decode: the input on the 1/4096 grid, S exact against the
    oracle's palettes, r = the float32 square root of S rounded to float32,
    r_x + r_y summed exactly in float64."""
    lab = ref["labels"].reshape(-1)
    sel = lab > 0
    Dch = emb.shape[-1]
    v = np.clip(emb.reshape(-1, Dch)[sel].astype(np.float32), -1.5, 1.5)
    X = np.rint(np.float32(4096.0) * v).astype(np.int64)
    k = lab[sel] - 1
    a, b = ref["centroids"]["bin_x"][k], ref["centroids"]["bin_y"][k]

    def dist(Xa, P):
        S = ((Xa - P.astype(np.int64)) ** 2).sum(-1)
        return np.sqrt(S.astype(np.float32)).astype(np.float64)

    return dist(X[:, :2 * F], ref["pal_x"][a]) + dist(X[:, Dch // 2:Dch // 2 + 2 * F], ref["pal_y"][b])


def run_ex(dec, emb, fg, fg_thr, theta, tau):
    e = torch.from_numpy(np.ascontiguousarray(emb)).cuda()
    g = None if fg is None else torch.from_numpy(np.ascontiguousarray(fg)).cuda()
    res = dec.run(e, g, fg_thr, theta, score=True, tau=tau)
    hist = torch.empty((dec.bins_h, dec.bins_w), dtype=torch.int64, device="cuda")
    assert dec.histogram(hist) == 0
    torch.cuda.synchronize()
    res["hist"] = hist.cpu().numpy().view(np.uint64)
    return res


def _workload(cfg, bins=None):
    spec = synth.CONFIGS[cfg]
    if bins is None:
        th = thresholds()[str(cfg)]
    else:
        with open(GOLDEN) as fh:
            th = json.load(fh)["sweep"][str(bins)]
    return spec, th, synth.make_frame(cfg), bins or spec.bins


# (workload, bins or None for its own grid): matrix-core f32 and f16, generic
@pytest.mark.parametrize("cfg,bins", [(1, None), (2, None), (5, 64)])
def test_mask_threshold_parity(cfg, bins):
    spec, th, f, b = _workload(cfg, bins)
    fx, fy = spec.freqs()
    cap = th["capacity"]
    base = oracle.decode(f.emb, f.fg, fx, fy, b, b, cap, spec.fg_threshold, th["peak_threshold"])
    D = np.sort(code_sums(base, f.emb, spec.n_freq))
    np.testing.assert_allclose(np.exp(-D / 4096.0), np.sort(base["score_map"][base["labels"] > 0])[::-1], rtol=1e-6)
    taus = [0.0, D[len(D) // 3] / 4096.0, (D[len(D) // 2] + 0.5) / 4096.0, D[(3 * len(D)) // 4] / 4096.0, math.inf]
    dec = native().Decoder(spec.H, spec.W, spec.n_freq, spec.dtype, fx, fy, b, b, cap)
    for tau in taus:
        print(f"config {cfg} bins {b} tau {tau}", flush=True)
        ref = oracle.decode(f.emb, f.fg, fx, fy, b, b, cap, spec.fg_threshold, th["peak_threshold"], tau=tau)
        got = run_ex(dec, f.emb, f.fg, spec.fg_threshold, th["peak_threshold"], tau)
        assert_parity(got, ref, cap)
        if 0.0 < tau < math.inf:
            on = int((D == tau * 4096.0).sum())
            kept = int((got["labels"] > 0).sum())
            assert 0 < kept < (base["labels"] > 0).sum()
            assert kept == int((D < tau * 4096.0).sum()), (kept, on)
        if tau == 0.0:
            assert not got["labels"].any() and not got["centroids"]["npix"].any()
    dec.close()


@pytest.mark.parametrize("cfg,bins", [(1, None), (2, None), (5, 64)])
def test_all_pixels_parity(cfg, bins):
    spec, th, f, b = _workload(cfg, bins)
    fx, fy = spec.freqs()
    cap = th["capacity"]
    ref0 = oracle.decode(f.emb, None, fx, fy, b, b, cap, 0.0, 0.0)
    theta = 0.1 * ref0["hist"].max() * 2.0 ** -30
    dec = native().Decoder(spec.H, spec.W, spec.n_freq, spec.dtype, fx, fy, b, b, cap)
    for tau in (math.inf, 1.0):
        print(f"config {cfg} bins {b} all pixels tau {tau}", flush=True)
        ref = oracle.decode(f.emb, None, fx, fy, b, b, cap, 0.0, theta, tau=tau)
        got = run_ex(dec, f.emb, None, 0.0, theta, tau)
        assert ref["K"] >= 1
        assert_parity(got, ref, cap)
        if tau == math.inf:
            assert np.all(got["labels"] > 0)
    dec.close()


@pytest.mark.parametrize("case", [(48, 64, 4, np.float32, 16, 16, 64), (37, 29, 3, np.float16, 12, 10, 30),
                                  (70, 70, 8, np.float16, 64, 64, 1024)])
def test_ragged_frames_with_options(case):
    H, W, F, dt, bw, bh, cap = case
    rng = np.random.default_rng(H * W)
    emb, fg, fx, fy = _random_frame(rng, H, W, F, dt)
    ref0 = oracle.decode(emb, fg, fx, fy, bw, bh, cap, 0.5, 0.0)
    theta = 0.05 * ref0["hist"].max() * 2.0 ** -30
    base = oracle.decode(emb, fg, fx, fy, bw, bh, cap, 0.5, theta)
    D = np.sort(code_sums(base, emb, F))
    dec = native().Decoder(H, W, F, "f32" if dt == np.float32 else "f16", fx, fy, bw, bh, cap)
    for use_fg, tau in ((True, D[len(D) // 2] / 4096.0), (False, math.inf), (False, D[len(D) // 4] / 4096.0)):
        g = fg if use_fg else None
        ref = oracle.decode(emb, g, fx, fy, bw, bh, cap, 0.5, theta, tau=tau)
        got = run_ex(dec, emb, g, 0.5, theta, tau)
        assert_parity(got, ref, cap)
    dec.close()


def test_decode_ex_defaults_equal_decode():
    spec, th, f, b = _workload(0)
    fx, fy = spec.freqs()
    dec = native().Decoder(spec.H, spec.W, spec.n_freq, spec.dtype, fx, fy, b, b, th["capacity"])
    a = gpu_decode(dec, f.emb, f.fg, spec.fg_threshold, th["peak_threshold"])
    e = run_ex(dec, f.emb, f.fg, spec.fg_threshold, th["peak_threshold"], math.inf)
    assert a["K"] == e["K"] and np.array_equal(a["centroids"], e["centroids"])
    assert np.array_equal(a["labels"], e["labels"]) and np.array_equal(a["score_map"], e["score_map"])
    assert np.array_equal(a["hist"], e["hist"])
    dec.close()


# --------------------------------------------------------------------------
# binary masks
# --------------------------------------------------------------------------
def _masks(dec, labels_dev, first, count, H, W):
    m = torch.full((count * H * W,), 7, dtype=torch.uint8, device="cuda")   # poison: every byte must be written
    assert dec.masks(labels_dev, first, count, m) == 0
    torch.cuda.synchronize()
    return m.cpu().numpy().reshape(count, H, W)


@pytest.mark.parametrize("cfg", [1, 3])
def test_masks_from_workload_labels(cfg):
    spec = synth.CONFIGS[cfg]
    th = thresholds()[str(cfg)]
    f = synth.make_frame(cfg)
    fx, fy = spec.freqs()
    cap = th["capacity"]
    dec = native().Decoder(spec.H, spec.W, spec.n_freq, spec.dtype, fx, fy, spec.bins, spec.bins, cap)
    out = dec.new_outputs(score=False)
    e = torch.from_numpy(f.emb).cuda()
    g = torch.from_numpy(f.fg).cuda()
    assert dec.decode(e, g, spec.fg_threshold, th["peak_threshold"], out["centroids"], out["num_centroids"],
                      out["labels"]) == 0
    torch.cuda.synchronize()
    lab = out["labels"].cpu().numpy()
    K = int(out["num_centroids"].item())
    Kc = min(K, cap)
    print(f"config {cfg}: K {K}", flush=True)
    # every centroid's mask, then a sub-range that runs past K (empty masks)
    for first, count in ((0, Kc), (max(Kc - 3, 0), min(8, cap - max(Kc - 3, 0)))):
        m = _masks(dec, out["labels"], first, count, spec.H, spec.W)
        want = lab[None] == (first + 1 + np.arange(count))[:, None, None]
        assert np.array_equal(m, want.astype(np.uint8))
    if cfg == 1:    # against the oracle's labels too (the decode is bit-exact with them)
        ref = oracle.decode(f.emb, f.fg, fx, fy, spec.bins, spec.bins, cap, spec.fg_threshold, th["peak_threshold"],
                            want_score=False)
        m = _masks(dec, out["labels"], 0, Kc, spec.H, spec.W)
        assert np.array_equal(m, (ref["labels"][None] == np.arange(1, Kc + 1)[:, None, None]).astype(np.uint8))
        for k in range(Kc):
            assert int(m[k].sum()) == int(ref["centroids"]["npix"][k])
    dec.close()


@pytest.mark.parametrize("H,W", [(37, 29), (1, 1), (16, 1), (3, 100)])
def test_masks_ragged_sizes(H, W):
    rng = np.random.default_rng(H + W)
    cap = 20
    fx = np.array([2 * math.pi / W])
    fy = np.array([2 * math.pi / H])
    dec = native().Decoder(H, W, 1, "f32", fx, fy, 8, 5, cap)
    lab = rng.integers(0, cap + 2, size=(H, W)).astype(np.int32)    # any int32 values, also past cap
    ld = torch.from_numpy(lab).cuda()
    for first, count in ((0, cap), (5, 3), (19, 1)):
        m = _masks(dec, ld, first, count, H, W)
        assert np.array_equal(m, (lab[None] == (first + 1 + np.arange(count))[:, None, None]).astype(np.uint8))
    dec.close()


def test_option_and_mask_argument_errors():
    nat = native()
    spec = synth.CONFIGS[0]
    th = thresholds()["0"]
    fx, fy = spec.freqs()
    cap = th["capacity"]
    dec = nat.Decoder(spec.H, spec.W, spec.n_freq, spec.dtype, fx, fy, 32, 32, cap)
    out = dec.new_outputs(score=True)
    e = torch.zeros((spec.H, spec.W, spec.D), dtype=torch.float32, device="cuda")
    g = torch.zeros((spec.H, spec.W), dtype=torch.float32, device="cuda")
    args = (out["centroids"], out["num_centroids"], out["labels"], out["score_map"])
    bad = nat.CPE_ERR_INVALID_ARG
    assert dec.decode_ex(e, g, 0.5, 0.0, float("nan"), *args) == bad
    assert dec.decode_ex(e, g, 0.5, 0.0, -math.inf, *args) == bad
    assert dec.decode_ex(e, g, math.nan, 0.0, 1.0, *args) == bad
    assert dec.decode_ex(e, g, 0.5, math.inf, 1.0, *args) == bad
    assert dec.decode_ex(e, g, 0.5, 0.0, 1.0, *args, reserved=1) == bad
    assert dec.decode_ex(e, g, 0.5, 0.0, -5.0, *args) == 0           # negative tau: nothing labelled
    assert dec.decode_ex(e, None, 0.5, 0.0, math.inf, *args) == 0     # no foreground channel
    assert dec.decode(e, None, 0.5, 0.0, *args) == bad                 # cpe_decode needs one
    lab = out["labels"]
    m = torch.empty((cap + 1) * spec.H * spec.W + 16, dtype=torch.uint8, device="cuda")
    assert dec.masks(lab, 0, 0, m) == bad
    assert dec.masks(lab, -1, 2, m) == bad
    assert dec.masks(lab, cap - 1, 2, m) == bad
    assert dec.masks(lab, 0, 1, m[1:]) == bad                          # misaligned masks
    assert dec.masks(lab, 0, 1, m, H=spec.H + 1) == bad
    assert dec.masks(lab, 0, cap, m) == 0
    torch.cuda.synchronize()
    dec.close()


def test_far_pixels():
    """Foreground pixels far from every candidate (squared distances far
    above 2^24, where fl32(S) rounds; distances near the largest the input
    range allows): labels, counts and scores equal the oracle's, with no mask
    threshold and with tau on either side of some of their distance sums."""
    from tests import farframe
    emb, fg, fx, fy, theta, far = farframe.make()
    dec = native().Decoder(farframe.H, farframe.W, farframe.F, "f32", fx, fy, farframe.BINS, farframe.BINS,
                           farframe.CAP)
    for tau in (math.inf, 20.0, 100.0):
        print(f"far pixels tau {tau}", flush=True)
        ref = oracle.decode(emb, fg, fx, fy, farframe.BINS, farframe.BINS, farframe.CAP, 0.5, theta, tau=tau)
        got = run_ex(dec, emb, fg, 0.5, theta, tau)
        assert_parity(got, ref, farframe.CAP)
        if tau == 20.0:     # some far pixels below tau, some above
            lab = got["labels"].reshape(-1)[far]
            assert 0 < int((lab > 0).sum()) < len(far)
    dec.close()


@pytest.mark.parametrize("bins,fail", [(32, 0), (32, 1), (32, 2), (48, 0), (48, 1), (48, 2)])
def test_decode_after_a_failed_one_matches_the_oracle(bins, fail):
    """A decode that stops before one of its launches (the test hook reports
    it as a failed launch, CPE_ERR_HIP, after enqueueing the launches before
    it) leaves nothing behind: the next decode on the same handle, of another
    frame, equals the oracle bit for bit.  Matrix-core and generic kernels."""
    nat = native()
    spec = synth.CONFIGS[1]
    fx, fy = spec.freqs()
    frames = [synth.make_frame(1, i) for i in range(3)]
    theta = thresholds()["1"]["peak_threshold"] * (bins / 32.0) ** -2
    cap = ((bins + 1) // 2) ** 2
    dec = nat.Decoder(spec.H, spec.W, spec.n_freq, spec.dtype, fx, fy, bins, bins, cap)
    print(f"bins {bins}, failure before launch {fail}", flush=True)
    first = gpu_decode(dec, frames[0].emb, frames[0].fg, spec.fg_threshold, theta)
    assert first["K"] > 0
    e = torch.from_numpy(frames[1].emb).cuda()
    g = torch.from_numpy(frames[1].fg).cuda()
    out = dec.new_outputs(score=True)
    assert dec.test_fail_launch(fail) == 0
    st = dec.decode(e, g, spec.fg_threshold, theta, out["centroids"], out["num_centroids"], out["labels"],
                    out["score_map"])
    assert st == nat.CPE_ERR_HIP
    torch.cuda.synchronize()
    got = gpu_decode(dec, frames[2].emb, frames[2].fg, spec.fg_threshold, theta)
    ref = oracle.decode(frames[2].emb, frames[2].fg, fx, fy, bins, bins, cap, spec.fg_threshold, theta)
    assert ref["K"] > 0
    assert_parity(got, ref, cap)
    assert dec.test_fail_launch(3) == nat.CPE_ERR_INVALID_ARG
    dec.close()


def test_launch_count_and_stage_events():
    """Frames of up to 2^21 pixels on grids up to 32 x 32 take two launches
    (the vote launch compacts): stage events 0 and 1 are recorded back to
    back, 2-3 and 4-5 bracket the two kernels; larger grids and frames take
    three.  The decode with events on still equals the oracle."""
    import bench
    nat = native()
    spec = synth.CONFIGS[1]
    fx, fy = spec.freqs()
    th = thresholds()["1"]
    f = synth.make_frame(1)
    for bins, launches in ((32, 2), (48, 3)):
        theta = th["peak_threshold"] * (bins / 32.0) ** -2
        cap = ((bins + 1) // 2) ** 2
        dec = nat.Decoder(spec.H, spec.W, spec.n_freq, spec.dtype, fx, fy, bins, bins, cap)
        assert dec.launch_count() == launches
        assert [i for _, i in nat.stage_layout(dec)] == ([1, 2] if launches == 2 else [0, 1, 2])
        ev = bench.HipEvents(nat.STAGE_EVENTS)
        assert dec.set_stage_events(ev.ev) == 0
        got = gpu_decode(dec, f.emb, f.fg, spec.fg_threshold, theta)
        ms = [ev.elapsed_ms(2 * i, 2 * i + 1) for i in range(3)]
        assert dec.set_stage_events(None) == 0
        ev.close()
        print(f"bins {bins}: {launches} launches, stage ms {ms}", flush=True)
        assert ms[1] > 0 and ms[2] > 0
        if launches == 2:
            assert ms[0] < ms[1]          # no kernel between events 0 and 1
        else:
            assert ms[0] > 0
        ref = oracle.decode(f.emb, f.fg, fx, fy, bins, bins, cap, spec.fg_threshold, theta)
        assert_parity(got, ref, cap)
        dec.close()
    fx1 = np.array([2 * math.pi / 2048])
    big = nat.Decoder(1025, 2048, 1, "f16", fx1, fx1, 32, 32)      # 2,099,200 pixels > 2^21
    assert big.launch_count() == 3
    big.close()
