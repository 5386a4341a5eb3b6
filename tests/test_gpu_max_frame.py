"""The largest frame the library accepts: 32768 x 65280 = 2^31 - 2^23 pixels.

Every pixel carries the same embedding (the sin/cos encoding of the centre of
bin (16, 16), one harmonic per axis, fp16) and is foreground, so each pixel
adds the same rank-1 vote q_x(a) q_y(b) (Eq6/Eq11) and the whole histogram is
N times one pixel's vote.  One pixel's vote comes from the oracle on a small
frame with the same palettes: its extents are the full extents divided by 256
(x) and 4096 (y) and its frequencies the full ones times those factors, so
every bin-centre phase (Eq9) is the same fp64 number (scaling by a power of
two commutes with rounding).  The CPU test checks that the two palettes are
equal; the GPU test then checks the decode of the full frame through the C
ABI: the histogram equals N times the oracle's per-pixel vote exactly (every
pixel counted once), one centroid at bin (16, 16) holding all N pixels, and
label 1 everywhere.
"""
import math

import numpy as np
import pytest

import oracle

H, W = 32768, 65280                # H * W = 2^31 - 2^23, the documented maximum
SY, SX = 4096, 256                  # the small frame: 8 x 255 pixels
BINS, A, B = 32, 16, 16
N = H * W


def frequencies(h, w):
    return np.array([math.pi / w]), np.array([math.pi / h])


def pixel_value():
    """The embedding of bin (A, B)'s centre, as the oracle places centres."""
    fx, fy = frequencies(H, W)
    cx = ((A + 1) * float(W)) / (BINS + 1)
    cy = ((B + 1) * float(H)) / (BINS + 1)
    return np.array([math.sin(fx[0] * cx), math.cos(fx[0] * cx), math.sin(fy[0] * cy), math.cos(fy[0] * cy)],
                    dtype=np.float16)


def small_frame_decode():
    fx, fy = frequencies(H, W)
    h, w = H // SY, W // SX
    emb = np.broadcast_to(pixel_value(), (h, w, 4)).copy()
    fg = np.ones((h, w), np.float16)
    return oracle.decode(emb, fg, fx * SX, fy * SY, BINS, BINS, 16, 0.5, 0.0, want_score=False), h * w


def test_scaled_frame_has_the_full_extents_palettes():
    """The small frame's palettes equal those of the full extents, which the
    oracle gives on 1 x 65280 and 32768 x 1 frames."""
    fx, fy = frequencies(H, W)
    small, _ = small_frame_decode()
    row = oracle.decode(np.zeros((1, W, 4), np.float16), np.zeros((1, W), np.float16), fx, fy, BINS, BINS, 16,
                        0.5, 0.0, want_score=False)
    col = oracle.decode(np.zeros((H, 1, 4), np.float16), np.zeros((H, 1), np.float16), fx, fy, BINS, BINS, 16,
                        0.5, 0.0, want_score=False)
    assert np.array_equal(small["pal_x"], row["pal_x"])
    assert np.array_equal(small["pal_y"], col["pal_y"])
    # one strict maximum, at the encoded bin
    assert small["K"] == 1
    c = small["centroids"][0]
    assert (c["bin_x"], c["bin_y"]) == (A, B)


@pytest.mark.gpu
def test_largest_frame_counts_every_pixel_once():
    torch = pytest.importorskip("torch")
    from tests.test_gpu_parity import native
    small, n_small = small_frame_decode()
    hs = small["hist"].astype(object)
    per_pixel = hs // n_small
    assert np.all(per_pixel * n_small == hs)          # identical pixels: the small histogram is n_small x one vote
    want = (per_pixel * N).astype(np.uint64)          # < 2^64: at most N x 2^30

    fx, fy = frequencies(H, W)
    print(f"largest frame: {H} x {W} f16 D=4, {N} pixels", flush=True)
    dec = native().Decoder(H, W, 1, "f16", fx, fy, BINS, BINS, 16)
    try:
        pal_x, pal_y, _ = dec.tables()
        assert np.array_equal(pal_x, small["pal_x"]) and np.array_equal(pal_y, small["pal_y"])
        emb = torch.from_numpy(pixel_value()).cuda().expand(N, 4).contiguous()
        fg = torch.ones(N, dtype=torch.float16, device="cuda")
        o = dec.new_outputs()
        assert dec.decode(emb, fg, 0.5, 0.0, o["centroids"], o["num_centroids"], o["labels"]) == 0
        hist = torch.empty((BINS, BINS), dtype=torch.int64, device="cuda")
        assert dec.histogram(hist) == 0
        torch.cuda.synchronize()
        lo, hi = torch.aminmax(o["labels"])
        assert (int(lo), int(hi)) == (1, 1)
        del emb, fg
        got = hist.cpu().numpy().view(np.uint64)
        assert np.array_equal(got, want)
        assert int(o["num_centroids"].item()) == 1
        c = o["centroids"].cpu().numpy().view(oracle.CENTROID_DTYPE)[0]
        s = small["centroids"][0]
        assert (c["bin_x"], c["bin_y"], c["npix"]) == (A, B, N)
        assert c["x"] == np.float32(s["x"] * SX) and c["y"] == np.float32(s["y"] * SY)
        assert c["score"] == float(want[B, A]) * 2.0 ** -30
    finally:
        dec.close()
