"""The operating-point fixture (tests/golden/operating_points.json, written by
tests/golden/make_operating_points.py with the CPU oracle alone): it names a threshold for every
reuse level of every workload, each threshold is what the script's bisection returns for its
recorded trail, and the oracle still gives the recorded sample reuse (a fixture left stale by
a change of the oracle fails here)."""
import json
import os

import numpy as np

import oracle
import synth

HERE = os.path.dirname(os.path.abspath(__file__))
with open(os.path.join(HERE, "golden", "operating_points.json")) as _fh:
    OPS = json.load(_fh)["workloads"]


def test_every_level_of_every_workload_has_a_threshold():
    for name, w in synth.configs.CONFIGS.items():
        if not w.reuse_targets:
            continue
        assert name in OPS, f"{name} missing from the operating points"
        assert [lv["target"] for lv in OPS[name]["levels"]] == list(w.reuse_targets)


def test_thresholds_follow_the_bisection_rule():
    """0 % is the literal gate at tau = 2; every other level's trail starts at the midpoint of
    [-1, 1], halves the bracket towards the target, and returns the candidate closest to it."""
    for name, op in OPS.items():
        for lv in op["levels"]:
            if lv["target"] == 0.0:
                assert lv["tau"] == 2.0 and not lv["bisection"]
                continue
            lo, hi = -1.0, 1.0
            for tau, rho in lv["bisection"]:
                assert tau == 0.5 * (lo + hi), f"{name}: {tau} is not the bracket's midpoint"
                if rho > lv["target"]:
                    lo = tau
                else:
                    hi = tau
            best = min(lv["bisection"], key=lambda tr: abs(tr[1] - lv["target"]))
            assert lv["tau"] == best[0] and abs(best[1] - lv["target"]) <= 0.011
            assert float(np.float32(lv["tau"])) == lv["tau"], "thresholds are exact in float32"


def test_recorded_sample_reuse_is_reproduced_by_the_oracle():
    """ViT-B/16 (the cheapest workload): the oracle on the recorded sample groups at the
    recorded threshold gives the recorded weighted reuse rate."""
    op = OPS["vit_b16"]
    w = synth.get_config("vit_b16")
    m, G = w.model, w.group_size
    blob = synth.make_blob(m, w.weight_seed)
    lv = op["levels"][0]
    tot = 0.0
    for g0, gs, wt in op["sample_groups"]:
        assert gs == G
        fr = synth.render_frames(w.video, m.image_size, g0, G)
        r = oracle.encode(fr, blob, m.as_dict(), G, tau=lv["tau"])
        tot += wt * oracle.reuse_rate(r["masks"], G)
    assert abs(tot - lv["sample_reuse"]) < 1e-5
