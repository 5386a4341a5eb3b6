"""GPU parity: the HIP decoder (through the C ABI) against the CPU oracle.

Bit-exact on the vote histogram, the centroid records (bin indices, bin
centres, vote masses, pixel counts), the true centroid count and the label
map; the optional score map within 1e-5 relative.  Covers the five
workloads at full size with their frozen thresholds and the launch
configuration the benchmark uses, ragged and degenerate frames, every
harmonic count, both dtypes, small and large bin grids, capacity overflow,
empty foreground, non-finite inputs and repeat-decode determinism.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
from paper_2609_16874_amd import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "configs.json")


def thresholds():
    with open(GOLDEN) as fh:
        return json.load(fh)["configs"]


def native():
    from paper_2609_16874_amd import native as nat
    return nat


def gpu_decode(dec, emb, fg, fg_thr, theta, score=True):
    """One decode with the score map (the assignment's exact search) and,
    with score, a second one without it (labels only: the fast search that
    the benchmark runs), whose records and labels go to res["fast"]."""
    e = torch.from_numpy(np.ascontiguousarray(emb)).cuda()
    g = torch.from_numpy(np.ascontiguousarray(fg)).cuda()
    res = dec.run(e, g, fg_thr, theta, score=score)
    hist = torch.empty((dec.bins_h, dec.bins_w), dtype=torch.int64, device="cuda")
    assert dec.histogram(hist) == 0
    torch.cuda.synchronize()
    res["hist"] = hist.cpu().numpy().view(np.uint64)
    if score:
        fast = dec.run(e, g, fg_thr, theta, score=False)
        assert dec.histogram(hist) == 0
        torch.cuda.synchronize()
        fast["hist"] = hist.cpu().numpy().view(np.uint64)
        res["fast"] = fast
    return res


def assert_parity(got, ref, capacity, check_score=True):
    if "fast" in got:
        assert_parity(got["fast"], ref, capacity, check_score=False)
    assert got["K"] == ref["K"], (got["K"], ref["K"])
    assert np.array_equal(got["hist"], ref["hist"]), "vote histogram differs"
    assert len(got["centroids"]) == min(ref["K"], capacity)
    for f in ("bin_x", "bin_y", "npix", "reserved"):
        assert np.array_equal(got["centroids"][f], ref["centroids"][f]), f
    for f in ("x", "y", "score"):
        assert np.array_equal(got["centroids"][f], ref["centroids"][f]), f
        np.testing.assert_allclose(got["centroids"][f], ref["centroids"][f], rtol=1e-5)
    assert np.array_equal(got["labels"], ref["labels"]), f"labels differ at {np.argwhere(got['labels'] != ref['labels'])[:5]}"
    if check_score and "score_map" in got:
        np.testing.assert_allclose(got["score_map"], ref["score_map"], rtol=1e-5, atol=0)


def run_pair(emb, fg, fx, fy, bw, bh, cap, fg_thr, theta, dtype=None, dec=None):
    nat = native()
    H, W, D = emb.shape
    dtype = dtype or ("f32" if emb.dtype == np.float32 else "f16")
    own = dec is None
    if own:
        dec = nat.Decoder(H, W, D // 4, dtype, fx, fy, bw, bh, cap)
    got = gpu_decode(dec, emb, fg, fg_thr, theta)
    ref = oracle.decode(emb, fg, fx, fy, bw, bh, cap, fg_thr, theta)
    if own:
        dec.close()
    return got, ref


# --------------------------------------------------------------------------
# the five workloads at full size
# --------------------------------------------------------------------------
@pytest.mark.parametrize("cfg", [0, 1, 2, 3])
def test_workload_parity(cfg):
    spec = synth.CONFIGS[cfg]
    th = thresholds()[str(cfg)]
    f = synth.make_frame(cfg)
    fx, fy = spec.freqs()
    print(f"config {cfg}: {spec.name}", flush=True)
    got, ref = run_pair(f.emb, f.fg, fx, fy, spec.bins, spec.bins, th["capacity"], spec.fg_threshold,
                        th["peak_threshold"])
    assert ref["K"] >= 1
    assert_parity(got, ref, th["capacity"])


@pytest.mark.parametrize("bins", list(synth.SWEEP_BINS))
def test_paper_shape_bin_sweep_parity(bins):
    """The paper's own decoder shape (704x704, L = 4 harmonics, fp32) at every
    bin count of its Table 1 sweep, with the thresholds calibrated per grid:
    grids up to 32x32 take the matrix-core kernels, larger ones the generic
    kernels and the stand-alone peak kernel."""
    spec = synth.CONFIGS[5]
    with open(GOLDEN) as fh:
        th = json.load(fh)["sweep"][str(bins)]
    f = synth.make_frame(5)
    fx, fy = spec.freqs()
    print(f"config 5 {spec.name} bins {bins}", flush=True)
    got, ref = run_pair(f.emb, f.fg, fx, fy, bins, bins, th["capacity"], spec.fg_threshold, th["peak_threshold"])
    assert ref["K"] >= 1
    assert_parity(got, ref, th["capacity"])


def test_workload4_batch_back_to_back():
    """All 16 frames of the batch workload decoded back to back on one handle
    and one stream (the launch sequence the benchmark times), each frame's
    vote histogram copied out on the same stream right after its decode;
    every frame's histogram, records, K, labels and score map compared with
    the oracle."""
    nat = native()
    spec = synth.CONFIGS[4]
    th = thresholds()["4"]
    fx, fy = spec.freqs()
    dec = nat.Decoder(spec.H, spec.W, spec.n_freq, spec.dtype, fx, fy, spec.bins, spec.bins, th["capacity"])
    frames = [synth.make_frame(4, i) for i in range(spec.n_frames)]
    embs = [torch.from_numpy(fr.emb).cuda() for fr in frames]
    fgs = [torch.from_numpy(fr.fg).cuda() for fr in frames]
    # pass 0: labels only, as the benchmark decodes (the fast assignment
    # search); pass 1: with the score map (the exact search)
    runs = []
    for score in (False, True):
        outs = [dec.new_outputs(score=score) for _ in frames]
        hists = [torch.empty((spec.bins, spec.bins), dtype=torch.int64, device="cuda") for _ in frames]
        for i in range(len(frames)):
            o = outs[i]
            assert dec.decode(embs[i], fgs[i], spec.fg_threshold, th["peak_threshold"], o["centroids"],
                              o["num_centroids"], o["labels"], o["score_map"]) == 0
            assert dec.histogram(hists[i]) == 0
        runs.append((outs, hists))
    torch.cuda.synchronize()
    for i, fr in enumerate(frames):
        print(f"config 4 frame {i}", flush=True)
        ref = oracle.decode(fr.emb, fr.fg, fx, fy, spec.bins, spec.bins, th["capacity"], spec.fg_threshold,
                            th["peak_threshold"])
        for outs, hists in runs:
            K = int(outs[i]["num_centroids"].item())
            got = {"K": K, "centroids": outs[i]["centroids"].cpu().numpy().view(nat.CENTROID_DTYPE)[:min(K, dec.capacity)],
                   "labels": outs[i]["labels"].cpu().numpy(), "hist": hists[i].cpu().numpy().view(np.uint64)}
            if outs[i]["score_map"] is not None:
                got["score_map"] = outs[i]["score_map"].cpu().numpy()
            assert_parity(got, ref, th["capacity"])
    dec.close()


@pytest.mark.parametrize("cfg", [0, 1, 2, 3])
def test_fast_and_exact_assignment_searches(cfg):
    """Label-only decodes in every search mode: the fast search at any size,
    every tile sent down the path that near ties of the fast search take
    (recomputed with correctly rounded distances, exact search), and the
    default: all equal to the oracle."""
    nat = native()
    spec = synth.CONFIGS[cfg]
    th = thresholds()[str(cfg)]
    f = synth.make_frame(cfg)
    fx, fy = spec.freqs()
    dec = nat.Decoder(spec.H, spec.W, spec.n_freq, spec.dtype, fx, fy, spec.bins, spec.bins, th["capacity"])
    ref = oracle.decode(f.emb, f.fg, fx, fy, spec.bins, spec.bins, th["capacity"], spec.fg_threshold,
                        th["peak_threshold"])
    for mode in (2, 1, 0):
        print(f"config {cfg}: search mode {mode}", flush=True)
        assert dec.test_search_mode(mode) == 0
        got = gpu_decode(dec, f.emb, f.fg, spec.fg_threshold, th["peak_threshold"], score=False)
        assert_parity(got, ref, th["capacity"], check_score=False)
    dec.close()


def test_square_root_is_correctly_rounded_on_its_whole_domain():
    """The assignment's distance sqrt_cr(fl32(S)) equals the IEEE correctly
    rounded binary32 square root on every value it can receive (0 and every
    float in [1, 2^32)): exhaustive, on the device."""
    assert native().check_sqrt() == 0


def test_tables_match_oracle():
    spec = synth.CONFIGS[2]
    fx, fy = spec.freqs()
    dec = native().Decoder(spec.H, spec.W, spec.n_freq, spec.dtype, fx, fy, 32, 32)
    pal_x, pal_y, wt = dec.tables()
    ref = oracle.decode(np.zeros((spec.H, spec.W, spec.D), np.float16), np.zeros((spec.H, spec.W), np.float16),
                        fx, fy, 32, 32)
    assert np.array_equal(pal_x, ref["pal_x"]) and np.array_equal(pal_y, ref["pal_y"])
    assert np.array_equal(wt, ref["weights"])
    dec.close()


# --------------------------------------------------------------------------
# ragged, degenerate and extreme cases
# --------------------------------------------------------------------------
def _random_frame(rng, H, W, F, dtype, n_inst=5, sigma=0.1, fg_noise=0.05):
    fx = np.array([2 * math.pi * 2 ** k / W for k in range(F)])
    fy = np.array([2 * math.pi * 2 ** k / H for k in range(F)])
    inst = rng.integers(0, n_inst + 1, size=(H, W))
    cx, cy = rng.uniform(0, W, n_inst + 1), rng.uniform(0, H, n_inst + 1)
    emb = synth.encode_positions(cx[inst], cy[inst], fx, fy) + sigma * rng.standard_normal((H, W, 4 * F))
    emb[inst == 0] = sigma * rng.standard_normal(((inst == 0).sum(), 4 * F))
    fg = (inst > 0) + fg_noise * rng.standard_normal((H, W))
    return emb.astype(dtype), fg.astype(dtype), fx, fy


CASES = [
    # H, W, F, dtype, bins_w, bins_h, capacity
    (37, 53, 4, np.float32, 16, 16, 64),
    (1, 1, 1, np.float32, 1, 1, 1),
    (1, 300, 2, np.float16, 5, 3, 15),
    (300, 1, 3, np.float32, 3, 5, 15),
    (61, 67, 1, np.float16, 7, 9, 63),
    (64, 64, 3, np.float16, 32, 32, 256),
    (50, 70, 5, np.float32, 32, 8, 64),
    (33, 47, 7, np.float16, 12, 20, 240),
    (40, 40, 9, np.float32, 32, 32, 256),
    (45, 39, 12, np.float16, 24, 24, 144),
    (64, 96, 16, np.float16, 32, 32, 256),
    (64, 96, 16, np.float32, 32, 32, 256),
    (70, 70, 8, np.float16, 64, 64, 1024),
    (90, 90, 4, np.float32, 80, 80, 1600),
    (128, 128, 4, np.float16, 128, 128, 4096),
    (257, 129, 8, np.float16, 32, 32, 1),          # capacity overflow
    (130, 130, 2, np.float32, 2, 2, 4),
]


@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}x{c[1]}_F{c[2]}_{np.dtype(c[3]).name}_b{c[4]}x{c[5]}_cap{c[6]}" for c in CASES])
def test_shapes_and_bins(case):
    H, W, F, dt, bw, bh, cap = case
    rng = np.random.default_rng(CASES.index(case))
    emb, fg, fx, fy = _random_frame(rng, H, W, F, dt)
    ref0 = oracle.decode(emb, fg, fx, fy, bw, bh, cap, 0.5, 0.0)
    theta = 0.05 * ref0["hist"].max() * 2.0 ** -30
    got, ref = run_pair(emb, fg, fx, fy, bw, bh, cap, 0.5, theta)
    assert_parity(got, ref, cap)


def _misaligned(t):
    """A device copy of t whose data starts one element past a 16-byte boundary."""
    buf = torch.empty(t.numel() + 16, dtype=t.dtype, device="cuda")
    v = buf[1:1 + t.numel()].view(t.shape)
    v.copy_(t)
    assert v.data_ptr() % 16 != 0 and v.data_ptr() % t.element_size() == 0
    return v


# Frames whose vote launch lists the participating pixels itself, eight
# consecutive pixels per lane: 64-pixel slices (640 x 640) and 1024-pixel
# slices (frames above 2^20 pixels) for the vote, contiguous ranges for the
# assignment, ragged last slices and ranges, fp16 and fp32 foreground planes,
# 16-byte aligned (vector loads) or aligned to their element only (one load
# per pixel).
FG_CASES = [(640, 640, 4, np.float16, True), (1023, 1027, 4, np.float32, True), (1024, 1024, 4, np.float32, False),
            (1025, 1029, 3, np.float16, False), (1025, 1029, 3, np.float16, True)]


@pytest.mark.parametrize("case", FG_CASES, ids=[f"{c[0]}x{c[1]}_{np.dtype(c[3]).name}_{'shifted' if c[4] else 'aligned'}"
                                                for c in FG_CASES])
def test_foreground_plane_layouts(case):
    H, W, F, dt, shifted = case
    rng = np.random.default_rng(H * 7 + W)
    emb, fg, fx, fy = _random_frame(rng, H, W, F, dt)
    ref0 = oracle.decode(emb, fg, fx, fy, 32, 32, 256, 0.5, 0.0)
    theta = 0.05 * ref0["hist"].max() * 2.0 ** -30
    ref = oracle.decode(emb, fg, fx, fy, 32, 32, 256, 0.5, theta)
    assert ref["K"] > 0
    dec = native().Decoder(H, W, F, "f32" if dt == np.float32 else "f16", fx, fy, 32, 32, 256)
    print(f"{H}x{W} {np.dtype(dt).name} foreground {'shifted' if shifted else 'aligned'}", flush=True)
    e = torch.from_numpy(emb).cuda()
    g = torch.from_numpy(fg).cuda()
    if shifted:
        g = _misaligned(g)
    got = dec.run(e, g, 0.5, theta, score=True)
    hist = torch.empty((32, 32), dtype=torch.int64, device="cuda")
    assert dec.histogram(hist) == 0
    torch.cuda.synchronize()
    got["hist"] = hist.cpu().numpy().view(np.uint64)
    assert_parity(got, ref, 256)
    dec.close()


def test_no_centroid_and_empty_foreground():
    rng = np.random.default_rng(1)
    emb, fg, fx, fy = _random_frame(rng, 48, 40, 4, np.float32)
    got, ref = run_pair(emb, fg, fx, fy, 16, 16, 64, 0.5, 1e9)       # threshold above every bin
    assert ref["K"] == 0
    assert_parity(got, ref, 64)
    assert not got["labels"].any() and not got["score_map"].any()
    got, ref = run_pair(emb, np.zeros_like(fg), fx, fy, 16, 16, 64, 0.5, -1.0)   # nobody votes
    assert_parity(got, ref, 64)
    got, ref = run_pair(emb, np.ones_like(fg), fx, fy, 16, 16, 64, 0.5, 0.0)     # everybody votes
    assert_parity(got, ref, 64)


def test_non_finite_and_saturating_inputs():
    rng = np.random.default_rng(2)
    emb, fg, fx, fy = _random_frame(rng, 40, 44, 4, np.float16)
    flat = emb.reshape(-1)
    idx = rng.choice(flat.size, 200, replace=False)
    flat[idx[:50]] = np.nan
    flat[idx[50:100]] = np.inf
    flat[idx[100:150]] = -np.inf
    flat[idx[150:]] = 30000.0
    fg.reshape(-1)[:5] = np.nan
    got, ref = run_pair(emb, fg, fx, fy, 16, 16, 64, 0.5, 0.5)
    assert_parity(got, ref, 64)


def test_repeat_decodes_are_bitwise_identical():
    nat = native()
    f = synth.make_frame(1)
    spec = f.spec
    fx, fy = spec.freqs()
    dec = nat.Decoder(spec.H, spec.W, spec.n_freq, spec.dtype, fx, fy, 32, 32)
    e = torch.from_numpy(f.emb).cuda()
    g = torch.from_numpy(f.fg).cuda()
    first = dec.run(e, g, 0.5, 2.5)
    for _ in range(20):
        again = dec.run(e, g, 0.5, 2.5)
        assert again["K"] == first["K"]
        assert np.array_equal(again["centroids"], first["centroids"])
        assert np.array_equal(again["labels"], first["labels"])
        assert np.array_equal(again["score_map"], first["score_map"])
    dec.close()


def test_argument_errors_on_device():
    nat = native()
    dec = nat.Decoder(16, 16, 4, "f32", np.ones(4), np.ones(4), 8, 8, 16)
    e = torch.zeros((16, 16, 16), dtype=torch.float32, device="cuda")
    g = torch.zeros((16, 16), dtype=torch.float32, device="cuda")
    o = dec.new_outputs(score=True)
    args = [o["centroids"], o["num_centroids"], o["labels"], o["score_map"]]
    assert dec.decode(e, g, 0.5, 0.0, *args) == 0
    assert dec.decode(e, g, 0.5, 0.0, *args, H=15) == nat.CPE_ERR_INVALID_ARG
    assert dec.decode(e, g, float("nan"), 0.0, *args) == nat.CPE_ERR_INVALID_ARG
    assert dec.decode(e, g, 0.5, float("inf"), *args) == nat.CPE_ERR_INVALID_ARG
    e_off = torch.zeros(16 * 16 * 16 + 4, dtype=torch.float32, device="cuda")[1:1 + 16 * 16 * 16]
    assert dec.decode(e_off, g, 0.5, 0.0, *args) == nat.CPE_ERR_INVALID_ARG       # 4-byte aligned only
    assert dec.decode(e, g, 0.5, 0.0, None, *args[1:]) == nat.CPE_ERR_INVALID_ARG
    torch.cuda.synchronize()
    dec.close()


@pytest.mark.parametrize("H,W", [(1000, 1000), (1024, 1024), (1030, 1024)])
def test_vote_slice_dealings_of_large_frames(H, W):
    """The vote launch deals 64-pixel slices in turn below 4096 pixels per
    workgroup (1000 x 1000), with a rotation per round from there when the
    rounds are whole (1024 x 1024), else 1024-pixel slices (1030 x 1024):
    each equals the oracle."""
    rng = np.random.default_rng(H * 7 + W)
    emb, fg, fx, fy = _random_frame(rng, H, W, 1, np.float16)
    ref0 = oracle.decode(emb, fg, fx, fy, 8, 8, 16, 0.5, 0.0)
    theta = 0.05 * ref0["hist"].max() * 2.0 ** -30
    print(f"{H}x{W}", flush=True)
    got, ref = run_pair(emb, fg, fx, fy, 8, 8, 16, 0.5, theta)
    assert ref["K"] > 0
    assert_parity(got, ref, 16)


@pytest.mark.parametrize("H,W", [(1024, 2048), (1, 2097153)])
def test_frames_at_the_two_launch_limit(H, W):
    """The largest frame whose vote launch lists the pixels itself (2^21
    pixels, two launches) and one pixel more (the compaction launch first,
    three launches): both equal the oracle."""
    nat = native()
    rng = np.random.default_rng(H + W)
    emb, fg, fx, fy = _random_frame(rng, H, W, 1, np.float16)
    ref0 = oracle.decode(emb, fg, fx, fy, 8, 8, 16, 0.5, 0.0)
    theta = 0.05 * ref0["hist"].max() * 2.0 ** -30
    dec = nat.Decoder(H, W, 1, "f16", fx, fy, 8, 8, 16)
    assert dec.launch_count() == (2 if H * W <= 2 ** 21 else 3)
    print(f"{H}x{W}: {dec.launch_count()} launches", flush=True)
    got, ref = run_pair(emb, fg, fx, fy, 8, 8, 16, 0.5, theta, dec=dec)
    assert ref["K"] > 0
    assert_parity(got, ref, 16)
    dec.close()
