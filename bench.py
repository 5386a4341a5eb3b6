#!/usr/bin/env python3
"""Benchmark of the gfx950 centroid-encoding decoder (one GPU).

Workload (one "step"): 16 synthetic 640x640 frames, D = 64 fp16 channels
(16 harmonics per axis), 10-100 mixed ellipse/polygon instances each,
decoded back to back with one cpe_decode call per frame on one stream.
Inputs are resident in HBM before timing starts.  Prints one JSON line:

  value        decoded frames per second (whole job, one GPU)
  ms_per_step  wall time of one 16-frame step (hipEvents around K steps)
  roofline     the dominant kernel's algorithmic bytes per launch divided by
               its average duration (start and end events recorded by the
               kernel's own dispatch), against 8 TB/s HBM
  cpu_baseline the plain single-threaded CPU oracle on a bounded sample of
               the same frames (reported, not a target)
  extra        the 640x640 single frame and the 1024x2048 frame, with the
               fraction of the HBM roofline for embedding read + label write

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0      # MI355X HBM3E peak, GB/s
GOLDEN = os.path.join(ROOT, "tests", "golden", "configs.json")
TRAFFIC = os.path.join(ROOT, "profiles", "traffic.json")
STAGE_KERNEL = {"compact": "k_compact", "recover_vote": "k_vote_mfma", "compact_vote": "k_vote_mfma",
                "assign_label": "k_assign_mfma"}


def source_sha256():
    """Hash of the library sources, as recorded with the profiler byte counts."""
    import glob
    import hashlib
    h = hashlib.sha256()
    files = sorted(glob.glob(os.path.join(ROOT, "paper_2609_16874_amd", "csrc", "*.hpp")) +
                   glob.glob(os.path.join(ROOT, "paper_2609_16874_amd", "csrc", "*.hip")) +
                   glob.glob(os.path.join(ROOT, "include", "*.h")))
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload_tag, stage):
    """HBM bytes per launch of the stage's kernel from the committed profiler
    counts (FETCH_SIZE and WRITE_SIZE scaled by a copy calibration), or None
    when they are missing or were taken on different sources."""
    try:
        with open(TRAFFIC) as fh:
            t = json.load(fh)
        if t["source_sha256"] != source_sha256():
            return None
        # the kernel's entry, named with its variant where it has several
        # (one ran on the workload: "k_assign_mfma (exact search)")
        name = STAGE_KERNEL[stage]
        hits = [v for k, v in t["workloads"][workload_tag]["kernels"].items()
                if k == name or k.startswith(name + " (")]
        return hits[0]["bytes"] if len(hits) == 1 else None
    except (OSError, KeyError, ValueError):
        return None


def progress(msg):
    """A progress line on stderr (stdout carries only the JSON result)."""
    print(f"bench: {msg}", file=sys.stderr, flush=True)


def thresholds():
    with open(GOLDEN) as fh:
        return json.load(fh)["configs"]


class HipEvents:
    """Raw hipEvent_t handles (the library records them on the decode stream)."""

    def __init__(self, n):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.ev = (ctypes.c_void_p * n)()
        for i in range(n):
            h = ctypes.c_void_p()
            assert self.hip.hipEventCreate(ctypes.byref(h)) == 0
            self.ev[i] = h

    def elapsed_ms(self, i, j):
        out = ctypes.c_float()
        assert self.hip.hipEventSynchronize(self.ev[j]) == 0
        assert self.hip.hipEventElapsedTime(ctypes.byref(out), self.ev[i], self.ev[j]) == 0
        return out.value

    def close(self):
        for e in self.ev:
            self.hip.hipEventDestroy(e)


def load_workload(cfg, n_frames=None):
    import torch
    from paper_2609_16874_amd import synth
    spec = synth.CONFIGS[cfg]
    n = spec.n_frames if n_frames is None else n_frames
    frames = [synth.make_frame(cfg, i) for i in range(n)]
    embs = [torch.from_numpy(f.emb).cuda() for f in frames]
    fgs = [torch.from_numpy(f.fg).cuda() for f in frames]
    return spec, frames, embs, fgs


def frame_bytes(spec, frame):
    """Algorithmic bytes: literal (full embedding + labels), and what each
    kernel must move given the participating set S (fg > threshold)."""
    es = 2 if spec.dtype == "f16" else 4
    npx = spec.H * spec.W
    nfg = int((frame.fg.astype(np.float32) > np.float32(spec.fg_threshold)).sum())
    return {
        "literal": npx * spec.D * es + 4 * npx,
        "compact": npx * es + 4 * nfg + 4 * (npx - nfg),
        "recover_vote": 4 * nfg + nfg * spec.D * es,
        "compact_vote": npx * es + 4 * nfg + 4 * (npx - nfg) + nfg * spec.D * es,
        "assign_label": 4 * nfg + nfg * spec.D * es + 4 * nfg,
        "peaks_assign_label": npx * spec.D * es + npx * es + 4 * npx,
        "n_fg": nfg,
    }


def time_steps(dec, embs, fgs, outs, fg_thr, theta, steps, warmup, min_warm_ms=0.0):
    """ms per step over `steps` timed steps after `warmup` untimed ones (and,
    with min_warm_ms, further untimed steps until that much wall time has
    passed, so that the clocks have left their idle state)."""
    import torch

    def step():
        for i in range(len(embs)):
            o = outs[i]
            st = dec.decode(embs[i], fgs[i], fg_thr, theta, o["centroids"], o["num_centroids"], o["labels"])
            if st != 0:
                raise RuntimeError(f"cpe_decode failed with status {st}")

    w0 = time.perf_counter()
    done = 0
    while done < warmup or (time.perf_counter() - w0) * 1e3 < min_warm_ms:
        step()
        done += 1
        if done % 8 == 0:
            torch.cuda.synchronize()
    time_steps.warmup_done = done
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    h0 = time.perf_counter()
    for _ in range(steps):
        step()
    host_s = time.perf_counter() - h0
    t1.record()
    torch.cuda.synchronize()
    time_steps.host_us_per_call = host_s / (steps * len(embs)) * 1e6
    return t0.elapsed_time(t1) / steps


def step_latency(dec, embs, fgs, outs, fg_thr, theta, steps=100, warmup=10):
    """Per-frame latency distribution: each of `steps` steps (one decode per
    frame of the workload, back to back) bracketed by its own pair of events,
    after `warmup` untimed steps; ms per frame = step time / frames."""
    import torch
    nfr = len(embs)

    def step():
        for i in range(nfr):
            o = outs[i]
            assert dec.decode(embs[i], fgs[i], fg_thr, theta, o["centroids"], o["num_centroids"], o["labels"]) == 0

    for _ in range(warmup):
        step()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    for a, b in ev:
        a.record()
        step()
        b.record()
    torch.cuda.synchronize()
    t = np.array([a.elapsed_time(b) for a, b in ev]) / nfr
    return {"steps": steps, "warmup": warmup, "mean": round(float(t.mean()), 5), "std": round(float(t.std()), 5),
            "min": round(float(t.min()), 5), "p50": round(float(np.percentile(t, 50)), 5),
            "p99": round(float(np.percentile(t, 99)), 5)}


def copy_bandwidth(mib=256, reps=10):
    """GB/s (bytes read + bytes written) of a plain device-to-device copy on
    this GPU: its practical HBM ceiling beside the 8 TB/s peak."""
    import torch
    n = mib << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda").random_(0, 255)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for _ in range(reps):
        dst.copy_(src)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / reps
    del src, dst
    return 2 * n / (ms * 1e-3) / 1e9


def stage_times(dec, embs, fgs, outs, fg_thr, theta, reps):
    """Average duration of each of the frame's kernels over reps x frames,
    from the start and end events their dispatches record."""
    from paper_2609_16874_amd import native
    layout = native.stage_layout(dec)
    names = [n for n, _ in layout]
    ev = HipEvents(native.STAGE_EVENTS)
    assert dec.set_stage_events(ev.ev) == 0
    acc = np.zeros(len(names))
    n = 0
    for _ in range(reps):
        for i in range(len(embs)):
            o = outs[i]
            assert dec.decode(embs[i], fgs[i], fg_thr, theta, o["centroids"], o["num_centroids"], o["labels"]) == 0
            acc += [ev.elapsed_ms(2 * i, 2 * i + 1) for _, i in layout]
            n += 1
    dec.set_stage_events(None)
    ev.close()
    return dict(zip(names, (acc / n).tolist()))


def panoptic_quality(labels, inst):
    """PQ of a decoded label map against the generating instance map (0 =
    background in both): segments match when their IoU exceeds 0.5 (then
    uniquely); PQ = sum of matched IoUs / (TP + FP/2 + FN/2).  Host-side
    evaluation of the outputs on a synthetic frame, outside any timing."""
    labels = np.asarray(labels, dtype=np.int64)
    inst = np.asarray(inst, dtype=np.int64)
    K, N = int(labels.max()), int(inst.max())
    m = (inst > 0) | (labels > 0)
    cnt = np.bincount(inst[m] * (K + 1) + labels[m], minlength=(N + 1) * (K + 1)).reshape(N + 1, K + 1)
    inter = cnt[1:, 1:].astype(np.float64)
    ia, la = cnt[1:, :].sum(1), cnt[:, 1:].sum(0)
    iou = inter / np.maximum(ia[:, None] + la[None, :] - inter, 1)
    tp = iou > 0.5
    ntp = int(tp.sum())
    nfn, nfp = int((ia > 0).sum()) - ntp, int((la > 0).sum()) - ntp
    return {"pq": round(float(iou[tp].sum()) / max(ntp + 0.5 * nfp + 0.5 * nfn, 1e-9), 4),
            "tp": ntp, "fp": nfp, "fn": nfn}


def bench_config(cfg, steps, warmup, n_frames=None, bins=None, th=None, loaded=None, n_used=None, quality=False,
                 min_warm_ms=0.0):
    """Time workload cfg; n_used: decode only the first n_used harmonics of
    the same embedding (the resolved-harmonics decode).  quality: also the
    PQ of each frame's labels against its instance map.  min_warm_ms: keep
    warming up until that much wall time has passed (the secondary lines,
    which follow seconds of host-side frame synthesis)."""
    from paper_2609_16874_amd import native
    th = th or thresholds()[str(cfg)]
    spec, frames, embs, fgs = loaded or load_workload(cfg, n_frames)
    fx, fy = spec.freqs()
    nf = n_used or spec.n_freq
    nb = bins or spec.bins
    dec = native.Decoder(spec.H, spec.W, nf, spec.dtype, fx[:nf], fy[:nf], nb, nb, th.get("capacity"), D=spec.D)
    outs = [dec.new_outputs() for _ in frames]
    ms_step = time_steps(dec, embs, fgs, outs, spec.fg_threshold, th["peak_threshold"], steps, warmup, min_warm_ms)
    stages = stage_times(dec, embs, fgs, outs, spec.fg_threshold, th["peak_threshold"], max(1, min(steps, 10)))
    bench_config.latency = step_latency(dec, embs, fgs, outs, spec.fg_threshold, th["peak_threshold"])
    fb = [frame_bytes(spec, f) for f in frames]
    mean_bytes = {k: float(np.mean([b[k] for b in fb])) for k in fb[0]}
    ws = dec.workspace_bytes()
    if quality:
        q = [dict(panoptic_quality(o["labels"].cpu().numpy(), f.inst), K=int(o["num_centroids"].item()),
                  instances=int(f.kept.sum())) for o, f in zip(outs, frames)]
        mean_bytes["quality"] = q[0] if len(q) == 1 else {"pq_mean": round(float(np.mean([x["pq"] for x in q])), 4),
                                                          "K_mean": float(np.mean([x["K"] for x in q]))}
    dec.close()
    return spec, frames, ms_step, stages, mean_bytes, ws


def cpu_baseline(cfg, frames, budget_s=12.0):
    """The oracle on the step's frames in order, cycling through them until
    about budget_s seconds of CPU work are done (at least one decode)."""
    import oracle
    th = thresholds()[str(cfg)]
    spec = frames[0].spec
    fx, fy = spec.freqs()
    avail = sorted(os.sched_getaffinity(0))
    os.sched_setaffinity(0, {avail[0]})    # one core, as a single-threaded baseline
    try:
        done, t0 = 0, time.perf_counter()
        while time.perf_counter() - t0 < budget_s:
            f = frames[done % len(frames)]
            oracle.decode(f.emb, f.fg, fx, fy, spec.bins, spec.bins, th["capacity"], spec.fg_threshold,
                          th["peak_threshold"], want_score=False)
            done += 1
        dt = time.perf_counter() - t0
    finally:
        os.sched_setaffinity(0, set(avail))
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            model = next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")), model)
    except OSError:
        pass
    return {"value": done / dt, "unit": "frames/s", "cores": 1, "kind": "oracle",
            "pinned_core": avail[0], "host_cpu": model, "host_cores_available": len(avail),
            "host_cores_total": os.cpu_count(),
            "sample": f"{done} decodes cycling through the {len(frames)} frames of the {spec.name} batch, "
                      f"single-threaded C oracle, {dt:.1f} s"}


def naive_ablation(cfg, reps=3):
    """The per-tuple ablation (cpe_decode_naive: per-(pixel, bin) float
    atomics and per-(pixel, candidate) aggregation, Table 3's "Naive") on
    frame 0 of workload cfg, timed like a step, beside the decoder on the same
    frame; and how many histogram bins differ bit for bit between two of its
    runs (float atomics add in a different order each time)."""
    import torch
    from paper_2609_16874_amd import native
    th = thresholds()[str(cfg)]
    spec, frames, embs, fgs = load_workload(cfg, 1)
    fx, fy = spec.freqs()
    dec = native.Decoder(spec.H, spec.W, spec.n_freq, spec.dtype, fx, fy, spec.bins, spec.bins, th["capacity"])
    o = dec.new_outputs()
    hist = torch.empty((spec.bins, spec.bins), dtype=torch.float32, device="cuda")

    def run():
        st = dec.decode_naive(embs[0], fgs[0], spec.fg_threshold, th["peak_threshold"], o["centroids"],
                              o["num_centroids"], o["labels"], hist)
        if st != 0:
            raise RuntimeError(f"cpe_decode_naive failed with status {st}")

    run()
    torch.cuda.synchronize()
    first = hist.clone()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(reps):
        run()
    t1.record()
    torch.cuda.synchronize()
    naive_ms = t0.elapsed_time(t1) / reps
    differ = int((hist.view(torch.int32) != first.view(torch.int32)).sum().item())
    opt_ms = time_steps(dec, embs, fgs, [dec.new_outputs()], spec.fg_threshold, th["peak_threshold"], 10, 3)
    dec.close()
    return {"workload": spec.name, "naive_ms_per_frame": round(naive_ms, 3), "decoder_ms_per_frame": round(opt_ms, 5),
            "naive_over_decoder": round(naive_ms / opt_ms, 1), "hist_bins_differing_between_naive_runs": differ,
            "bins": spec.bins * spec.bins}


# The paper's optimised decoder latency for its 704x704, L = 4 maps on a Jetson
# Orin Nano in fp32 (Table 1), by bin count: context only, other hardware.
PAPER_TABLE1_MS = {8: 2.13, 16: 6.13, 32: 30.66, 64: 101.37, 80: 144.00}


def sweep(steps, warmup):
    """Bin-count sweep (Table 1's grids) on workload 5, the paper's own
    decoder shape, and the resolution series of every workload at 32x32."""
    from paper_2609_16874_amd import synth
    with open(GOLDEN) as fh:
        sw = json.load(fh)["sweep"]
    out = {"bins_sweep": [], "resolution": []}
    loaded = load_workload(5)
    for b in synth.SWEEP_BINS:
        th = sw[str(b)]
        progress(f"sweep: {b}x{b} bins")
        s, fr, ms, st, by, ws = bench_config(5, steps, warmup, bins=b, th=th, loaded=loaded, min_warm_ms=150.0)
        out["bins_sweep"].append({"workload": s.name, "bins": b, "ms_per_frame": round(ms, 5),
                                  "frames_per_s": round(1000.0 / ms, 1), "workspace_bytes": ws,
                                  "path": "matrix-core" if b <= 32 else "matrix-core vote, generic assignment",
                                  "stages_ms": {k: round(v, 5) for k, v in st.items()},
                                  "paper_ms_orin_nano_fp32": PAPER_TABLE1_MS[b]})
    del loaded
    for cfg in sorted(synth.CONFIGS):
        progress(f"resolution series: workload {cfg}")
        s, fr, ms, st, by, ws = bench_config(cfg, steps, warmup, min_warm_ms=150.0)
        nfr = len(fr)
        out["resolution"].append({"workload": s.name, "pixels": s.H * s.W, "D": s.D, "dtype": s.dtype,
                                  "ms_per_frame": round(ms / nfr, 5), "frames_per_s": round(nfr * 1000.0 / ms, 1),
                                  "literal_roofline_frac": round(by["literal"] / (ms / nfr * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                                  "workspace_bytes": ws})
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--no-extra", action="store_true", help="skip the single-frame 640x640 and 1024x2048 lines")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU-oracle baseline")
    ap.add_argument("--only-config", type=int, default=None,
                    help="time only this config (0-4) and print its per-stage line; for profiler runs")
    ap.add_argument("--copy-calibration", type=int, default=None, metavar="MIB",
                    help="time a plain device copy of MIB MiB instead (reference for profiler byte counters)")
    ap.add_argument("--sweep", action="store_true",
                    help="bin-count sweep at the paper's 704x704 D=16 shape and the resolution series instead")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the decoder has no multi-GPU path (frames are independent "
              "and would shard across GPUs without communication; one GPU's throughput is what is measured)",
              file=sys.stderr)
        sys.exit(2)
    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"

    if args.copy_calibration is not None:
        n = args.copy_calibration << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").random_(0, 255)
        dst = torch.empty_like(src)
        for _ in range(args.warmup):
            dst.copy_(src)
        torch.cuda.synchronize()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record()
        for _ in range(args.steps):
            dst.copy_(src)
        t1.record()
        torch.cuda.synchronize()
        ms = t0.elapsed_time(t1) / args.steps
        print(json.dumps({"copy_bytes": n, "ms_per_copy": round(ms, 5),
                          "gbs_read_plus_write": round(2 * n / (ms * 1e-3) / 1e9, 1)}), flush=True)
        return
    if args.sweep:
        print(json.dumps(sweep(args.steps, args.warmup)), flush=True)
        return
    if args.only_config is not None:
        cfg = args.only_config
        s, fr, ms, st, b, ws = bench_config(cfg, args.steps, args.warmup, min_warm_ms=150.0)
        nfr = len(fr)
        print(json.dumps({"workload": s.name, "ms_per_frame": round(ms / nfr, 5),
                          "frames_per_s": round(nfr * 1000 / ms, 1), "literal_bytes": int(b["literal"]),
                          "literal_roofline_frac": round(b["literal"] / (ms / nfr * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                          "n_fg": int(b["n_fg"]), "stages_ms": {k: round(v, 5) for k, v in st.items()},
                          "ms_per_frame_stats": bench_config.latency,
                          "host_enqueue_us_per_frame": round(time_steps.host_us_per_call, 2),
                          "workspace_bytes": ws}), flush=True)
        return

    progress("16x640x640 workload")
    spec, frames, ms_step, stages, bytes_, ws = bench_config(4, args.steps, args.warmup)
    latency = bench_config.latency
    progress(f"16x640x640: {ms_step / len(frames):.5f} ms per frame")
    copy_gbs = copy_bandwidth()
    nfr = len(frames)
    fps = nfr * 1000.0 / ms_step
    dom = max(stages, key=stages.get)
    dom_ms = stages[dom]
    achieved = bytes_[dom] / (dom_ms * 1e-3) / 1e9
    traffic = measured_traffic("16x640x640", dom)
    literal_gbs = bytes_["literal"] / (ms_step / nfr * 1e-3) / 1e9
    result = {
        "metric": "decoded frames/sec at 640x640 D=64",
        "value": round(fps, 2),
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "ms_per_frame": round(ms_step / nfr, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {"workload": spec.name, "frames_per_step": nfr, "H": spec.H, "W": spec.W, "D": spec.D,
                   "input_dtype": spec.dtype, "bins": spec.bins, "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic,
                     "traffic_gbs": None if traffic is None else round(traffic / (dom_ms * 1e-3) / 1e9, 1),
                     "bytes_per_launch": round(bytes_[dom]), "avg_launch_ms": round(dom_ms, 5)},
        "stages_ms": {k: round(v, 5) for k, v in stages.items()},
        "ms_per_frame_stats": latency,
        "literal_roofline_frac": round(literal_gbs / HBM_PEAK_GBS, 4),
        "copy_gbs": round(copy_gbs, 1),
        "literal_frac_of_copy": round(literal_gbs / copy_gbs, 4),
        "host_enqueue_us_per_frame": round(time_steps.host_us_per_call, 2),
        "workspace_bytes": ws,
    }
    if not args.no_extra:
        from paper_2609_16874_amd import harmonics
        with open(GOLDEN) as fh:
            resolved = json.load(fh)["resolved"]
        extra = {}
        for cfg in (2, 3):
            progress(f"secondary workload {cfg}")
            loaded = load_workload(cfg)
            s, fr, ms, st, b, _ = bench_config(cfg, max(1, args.steps // 2), max(1, args.warmup // 2),
                                               loaded=loaded, quality=True, min_warm_ms=150.0)
            extra[f"cfg{cfg}"] = {"workload": s.name, "ms_per_frame": round(ms, 5), "frames_per_s": round(1000 / ms, 1),
                                  "literal_bytes": int(b["literal"]),
                                  "literal_roofline_frac": round(b["literal"] / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                                  "literal_frac_of_copy": round(b["literal"] / (ms * 1e-3) / 1e9 / copy_gbs, 4),
                                  "ms_per_frame_stats": bench_config.latency,
                                  "stages_ms": {k: round(v, 5) for k, v in st.items()},
                                  "quality_vs_instances": b["quality"]}
            if cfg == 3 and not args.no_cpu:      # one oracle decode of the frame, one core
                extra["cfg3"]["cpu_baseline"] = cpu_baseline(3, loaded[1], budget_s=0.1)
            # the same frame decoded with only the harmonics the 32x32 grid resolves
            fx, fy = s.freqs()
            n = harmonics.resolved_pair(fx, fy, s.W, s.H, s.bins, s.bins)
            th = dict(resolved[str(cfg)], capacity=thresholds()[str(cfg)]["capacity"])
            s, fr, ms, st, b, _ = bench_config(cfg, max(1, args.steps // 2), max(1, args.warmup // 2), th=th,
                                               loaded=loaded, n_used=n, quality=True, min_warm_ms=150.0)
            extra[f"cfg{cfg}_resolved"] = {"workload": s.name, "harmonics_decoded": n,
                                           "ms_per_frame": round(ms, 5), "frames_per_s": round(1000 / ms, 1),
                                           "stages_ms": {k: round(v, 5) for k, v in st.items()},
                                           "quality_vs_instances": b["quality"]}
            del fr, loaded
        # Table 3's naive-vs-optimised contrast on this GPU: the paper's own
        # shape (704x704, L = 4) and a 640x640 D = 64 frame
        progress("naive ablation")
        extra["naive_ablation"] = [naive_ablation(5), naive_ablation(2)]
        result["extra"] = extra
    if not args.no_cpu:
        progress("CPU oracle baseline")
        result["cpu_baseline"] = cpu_baseline(4, frames)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
