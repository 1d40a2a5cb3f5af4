"""Writes operating_points.json: the gate threshold of every reuse level the workloads name,
calibrated with the CPU oracle alone.

For each workload and target reuse rate the threshold tau is found by bisection on [-1, 1]
(midpoints only, so every candidate is a dyadic value that float32 holds exactly): the oracle
encodes a stratified sample of whole groups of the workload's video in gate mode, the sample's
reuse rate (the reuse-rate definition of the reuse-loss equation, Section 4: non-reference
frames, all tokens, all layers) is the strata's rates weighted by each stratum's share of the
workload's groups, and the bisection stops at the first tau within 0.01 of the target (else
keeps the closest).  A target of 0 is the literal gate with tau = 2 (no cosine reaches it), so
it needs no search.  The thresholds choose where the parity tests and the bench operate; they
are inputs, not expected values, and nothing here runs on the GPU.

Usage: python tests/golden/make_operating_points.py [workload ...]   (default: all)
"""
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth  # noqa: E402

OUT = os.path.join(HERE, "operating_points.json")

# Stratified samples: (first frame of a group, weight = that stratum's share of the groups).
SAMPLES = {
    # 64 frames, groups of 4, one static scene: four groups spread over the clip
    "vit_b16": [(0, 0.25), (16, 0.25), (32, 0.25), (48, 0.25)],
    # 256 frames, groups of 8, one panning scene: four groups spread over the batch
    "vit_l14": [(0, 0.25), (64, 0.25), (128, 0.25), (192, 0.25)],
    # 1024 frames, groups of 8, scene cuts at 60 + 120 k: 9 of the 128 groups hold a cut
    "vit_l14_336": [(0, 59.5 / 128), (64, 59.5 / 128), (56, 9 / 128)],
    # 7200 frames, groups of 8, a 240-frame cycle of 120 static, 80 panning and 40 busy frames
    # (15, 10 and 5 groups of each cycle's 30)
    "vit_h14": [(0, 15 / 30), (120, 10 / 30), (200, 5 / 30)],
}
NO_REUSE_TAU = 2.0


def sample_reuse(w, blob, frames, tau):
    m, G = w.model, w.group_size
    tot = 0.0
    for (g0, wt) in SAMPLES[w.name]:
        r = oracle.encode(frames[g0], blob, m.as_dict(), G, tau=tau)
        tot += wt * oracle.reuse_rate(r["masks"], G)
    return tot


def calibrate(w, blob, frames, target, tol=0.01, iters=24):
    lo, hi, best, trail = -1.0, 1.0, None, []
    for _ in range(iters):
        mid = 0.5 * (lo + hi)
        rho = sample_reuse(w, blob, frames, mid)
        trail.append([mid, round(rho, 5)])
        print(f"  [{w.name}] target {target}: tau {mid!r} -> sample reuse {rho:.4f}", flush=True)
        if best is None or abs(rho - target) < abs(best[1] - target):
            best = (mid, rho)
        if abs(rho - target) <= tol:
            break
        if rho > target:
            lo = mid
        else:
            hi = mid
    return best, trail


def save(name, entry):
    """Read-modify-write of the fixture under a lock, so that workloads can run in parallel."""
    import fcntl
    import tempfile
    with open(os.path.join(tempfile.gettempdir(), "operating_points.lock"), "w") as lk:
        fcntl.flock(lk, fcntl.LOCK_EX)
        res = {}
        if os.path.exists(OUT):
            with open(OUT) as fh:
                res = json.load(fh)["workloads"]
        res[name] = entry
        with open(OUT, "w") as fh:
            json.dump({"about": "gate thresholds of the workloads' reuse levels, calibrated with "
                                "the CPU oracle on stratified samples of whole groups "
                                "(make_operating_points.py)",
                       "workloads": {k: res[k] for k in sorted(res)}}, fh, indent=1)


def main(names):
    for name in names:
        w = synth.get_config(name)
        m, G = w.model, w.group_size
        blob = synth.make_blob(m, w.weight_seed)
        frames = {g0: synth.render_frames(w.video, m.image_size, g0, G) for g0, _ in SAMPLES[name]}
        t0 = time.time()
        levels = []
        for tgt in w.reuse_targets:
            if tgt == 0.0:
                levels.append({"target": 0.0, "tau": NO_REUSE_TAU, "sample_reuse": 0.0,
                               "bisection": []})
                continue
            (tau, rho), trail = calibrate(w, blob, frames, tgt)
            levels.append({"target": tgt, "tau": tau, "sample_reuse": round(rho, 5),
                           "bisection": trail})
        save(name, {"sample_groups": [[g0, G, wt] for g0, wt in SAMPLES[name]],
                    "levels": levels, "cpu_seconds": round(time.time() - t0, 1)})
        print(f"[{name}] " + ", ".join(f"{lv['target']:.0%}: tau {lv['tau']!r}" for lv in levels),
              flush=True)


if __name__ == "__main__":
    main(sys.argv[1:] or list(SAMPLES))
