"""Write tests/golden/configs.json: the frozen peak threshold of each workload.

For workload c the threshold is 0.10 x the largest vote mass of the CPU
oracle's histogram on the calibration frame (seed [260916874, c, 999]), so
that a peak must collect at least a tenth of the strongest bin's votes; the
bin-count sweep of workload 5 gets one threshold per grid the same way, and
so does the resolved-harmonics decode of each workload (only the leading
harmonics its grid resolves, read from the same embedding).  Only the
generator, the harmonic-count rule and the oracle are called.  Run from the repository root:

    python -m tests.golden.make_configs
"""
import json
import os

import oracle
from paper_2609_16874_amd import harmonics, synth

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "configs.json")
FRACTION = 0.10


def main():
    out = {"fraction_of_max": FRACTION, "configs": {}}
    for c, spec in synth.CONFIGS.items():
        f = synth.make_frame(c, calibration=True)
        r = oracle.decode_frame(f, peak_threshold=0.0)
        hmax = int(r["hist"].max())
        out["configs"][str(c)] = {
            "name": spec.name, "bins": spec.bins, "fg_threshold": spec.fg_threshold,
            "capacity": ((spec.bins + 1) // 2) ** 2,
            "calibration_max_vote_mass": hmax * 2.0 ** -30,
            "peak_threshold": FRACTION * hmax * 2.0 ** -30,
        }
        print(c, out["configs"][str(c)])
    # workload 5 at every bin count of the sweep: its own calibration per grid
    out["sweep"] = {}
    f = synth.make_frame(5, calibration=True)
    for b in synth.SWEEP_BINS:
        r = oracle.decode_frame(f, bins=b, peak_threshold=0.0)
        hmax = int(r["hist"].max())
        out["sweep"][str(b)] = {"config": 5, "bins": b, "capacity": ((b + 1) // 2) ** 2,
                                "calibration_max_vote_mass": hmax * 2.0 ** -30,
                                "peak_threshold": FRACTION * hmax * 2.0 ** -30}
        print("sweep", b, out["sweep"][str(b)])
    # the resolved-harmonics decode: the first n harmonics of each axis block
    out["resolved"] = {}
    for c, spec in synth.CONFIGS.items():
        fx, fy = spec.freqs()
        n = harmonics.resolved_pair(fx, fy, spec.W, spec.H, spec.bins, spec.bins)
        f = synth.make_frame(c, calibration=True)
        r = oracle.decode(f.emb, f.fg, fx[:n], fy[:n], spec.bins, spec.bins, None, spec.fg_threshold, 0.0,
                          want_score=False)
        hmax = int(r["hist"].max())
        out["resolved"][str(c)] = {"config": c, "n_freq": n, "bins": spec.bins,
                                   "calibration_max_vote_mass": hmax * 2.0 ** -30,
                                   "peak_threshold": FRACTION * hmax * 2.0 ** -30}
        print("resolved", c, out["resolved"][str(c)])
    with open(OUT, "w") as fh:
        json.dump(out, fh, indent=1)


if __name__ == "__main__":
    main()
