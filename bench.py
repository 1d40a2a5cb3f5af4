"""Throughput of the reuse-aware ViT encoder on one MI355X.

Workload (default): ViT-L/14 at 224 px (257 tokens, depth 24, width 1024, 16 heads, MLP
4096, bf16 operands, fp32 accumulate), a batch of 256 synthetic video frames (6 moving
squares, 1 px/frame camera pan, pixel noise sigma 0.02) in groups of 8 frames.  The
reuse thresholds are the operating points for 50 %, 70 % and 90 % reuse calibrated with the
CPU oracle (tests/golden/operating_points.json).

One step = one encode of the batch at each of the three reuse levels (768 frames),
inputs already resident in device memory.  `value` = frames encoded per second over
the timed steps.  The line also carries each level's frames/s, the same kernels with
reuse off (tau = -inf) and the speedup over it, the roofline of the dominant kernel
(timed with HIP events on the encode stream over the timed region) against the nominal
peak and against the MFMA rate measured on the chip, and the CPU oracle timed on a bounded
sample of the same frames.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu]
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402

METRIC = "frames/s ViT-L/14 at 50/70/90% reuse; packed-GEMM MFMA util; speedup vs dense"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3    # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0

GEMM_STAGES = {"qkv": 3, "oproj": 1, "fc1": 4, "fc2": 4}   # Nout*K / D^2


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def active_rows(masks, G):
    """M_l per layer from a [F, L, N] reuse map (reference frames are fully recomputed)."""
    F, L, N = masks.shape
    act = (masks == 0)
    act[::G] = True
    return act.sum(axis=(0, 2))            # [L]


def reuse_of(masks, G):
    nonref = [f for f in range(masks.shape[0]) if f % G]
    return float((masks[nonref] != 0).mean()) if nonref else 0.0


def stage_flops(stage, m, Ml):
    """Algorithmic FLOPs of one launch of a stage at M_l active rows."""
    D, N = m.width, m.n_tokens
    if stage in ("qkv", "oproj"):
        return 2.0 * Ml * D * D * GEMM_STAGES[stage]
    if stage in ("fc1", "fc2"):
        return 2.0 * Ml * D * m.mlp
    if stage == "attn":
        return 4.0 * Ml * N * D
    return 0.0


def stage_bytes(stage, m, Ml):
    """Algorithmic HBM bytes of one launch of a GEMM stage at M_l active rows: bf16 operand rows
    and weights read once, fp32 residual rows read once, outputs written once, row indices."""
    D, Dm = m.width, m.mlp
    if stage == "qkv":
        return Ml * D * 2 + 3 * D * D * 2 + Ml * 3 * D * 2
    if stage == "oproj":
        return Ml * D * 2 + D * D * 2 + Ml * D * 4 + Ml * 4 + Ml * D * 4
    if stage == "fc1":
        return Ml * D * 2 + Dm * D * 2 + Ml * Dm * 2
    if stage == "fc2":
        return Ml * Dm * 2 + D * Dm * 2 + Ml * D * 4 + Ml * 4 + Ml * D * 4
    return 0.0


def attn_bytes(m, Ml, F):
    """Algorithmic HBM bytes of one attention launch: the packed query rows read and the output
    rows written once, and every frame's N keys and values (fresh or the reference's) once."""
    D, N = m.width, m.n_tokens
    return Ml * D * 2 * 2 + F * N * 2 * D * 2


def row_stage_bytes(stage, m, Ml_prev, Ml, F):
    """Algorithmic HBM bytes of one launch of a row kernel at layer l (Ml active rows, Ml_prev at
    the layer before; the whole batch at the first layer).  gate: the fp32 rows of every token not
    reused at the layer before (a token reused there holds its reference's row: cosine 1 without
    a read; reference frames are among the rows read), its LN1 row (bf16) for every recomputed
    token, and the map.  ln2: fp32 rows in, bf16 rows out.  compact: the map in, the packed row
    list and every token's packed slot out."""
    D, N = m.width, m.n_tokens
    if stage == "gate":
        return Ml_prev * D * 4 + Ml * D * 2 + F * N
    if stage == "ln2":
        return Ml * D * 4 + Ml * D * 2
    if stage == "compact":
        return F * N + Ml * 4 + F * N * 4 + (F + 1) * 4
    return 0.0


KERNEL_SOURCE = {"qkv": "gemm.hip", "oproj": "gemm.hip", "fc1": "gemm.hip", "fc2": "gemm.hip",
                 "patch": "gemm.hip", "attn": "attention.hip", "gate": "rowops.hip",
                 "ln2": "rowops.hip", "compact": "rowops.hip"}


def measured_traffic(stage, recorded_config):
    """HBM bytes per launch of `stage` from the committed counter record, if it was taken from
    the current kernel source and this run is the configuration it was taken on (the default
    ViT-L/14 sweep: `recorded_config`); else None."""
    import hashlib
    if not recorded_config:
        return None
    rec = os.path.join(ROOT, "profiles", f"{stage}_hbm_traffic.json")
    src = KERNEL_SOURCE.get(stage)
    if not src or not os.path.exists(rec):
        return None
    with open(rec) as fh:
        r = json.load(fh)
    path = os.path.join(ROOT, "paper_2506_14107_amd", "csrc", src)
    sha = hashlib.sha256(open(path, "rb").read()).hexdigest()
    return r["traffic_bytes_per_launch"] if r.get("source_sha256") == sha else None


STAGE_KERNEL = {"qkv": ("Epi)1",), "oproj": ("Epi)2",), "fc1": ("Epi)3",), "fc2": ("Epi)4",),
                "patch": ("Epi)0",),
                "attn": ("attn_unit_k", "attn_mfma_k", "attn_wave_k"), "gate": ("gate_k",),
                "ln2": ("ln_rows_k",), "compact": ("compact_k",)}   # name fragments per stage


def traffic_record(fetch_csv, write_csv, bench_json, cmds):
    """Turns two rocprofv3 --pmc passes over `bench.py --copy-calibration` (FETCH_SIZE, then
    WRITE_SIZE; KiB per dispatch) into profiles/<stage>_hbm_traffic.json for each stage.  The
    counters are scaled by what they read for the 1 GiB copy of the same run; the stage's
    launches of the timed region are the last ones before that copy."""
    import csv
    import hashlib
    bench = None
    with open(bench_json) as fh:
        for line in fh:
            if line.startswith("{"):
                bench = json.loads(line)
    stages = bench["stages"]

    def rows(path, counter):
        with open(path) as fh:
            rs = [r for r in csv.DictReader(fh) if r["Counter_Name"] == counter]
        rs.sort(key=lambda r: int(r["Dispatch_Id"]))
        copies = [r for r in rs if "copyBuffer" in r["Kernel_Name"] and int(r["Grid_Size"]) >= 131072]
        return rs, copies[-1]

    fr, fcopy = rows(fetch_csv, "FETCH_SIZE")
    wr, wcopy = rows(write_csv, "WRITE_SIZE")
    gib_kib = float(1 << 20)
    fs, ws = gib_kib / float(fcopy["Counter_Value"]), gib_kib / float(wcopy["Counter_Value"])
    out = {}
    for stage, info in stages.items():
        key, n = STAGE_KERNEL[stage], info["launches"]

        def timed(rs, cut):
            ks = [r for r in rs if any(k in r["Kernel_Name"] for k in key)
                  and int(r["Dispatch_Id"]) < cut]
            return ks[-n:]
        fk = timed(fr, int(fcopy["Dispatch_Id"]))
        wk = timed(wr, int(wcopy["Dispatch_Id"]))
        f_avg = float(np.mean([float(r["Counter_Value"]) for r in fk]))
        w_avg = float(np.mean([float(r["Counter_Value"]) for r in wk]))
        traffic = (f_avg * fs + w_avg * ws) * 1024
        src = os.path.join("paper_2506_14107_amd", "csrc", KERNEL_SOURCE[stage])
        sha = hashlib.sha256(open(os.path.join(ROOT, src), "rb").read()).hexdigest()
        rec = {"kernel": fk[0]["Kernel_Name"], "stage": stage, "source": src, "source_sha256": sha,
               "launches_averaged": len(fk), "fetch_kib_per_launch": round(f_avg, 1),
               "write_kib_per_launch": round(w_avg, 1),
               "copy_1GiB_fetch_kib": float(fcopy["Counter_Value"]),
               "copy_1GiB_write_kib": float(wcopy["Counter_Value"]),
               "fetch_scale": round(fs, 4), "write_scale": round(ws, 4),
               "traffic_bytes_per_launch": round(traffic),
               "algo_bytes_per_launch": info["algo_bytes_per_launch"],
               "traffic_over_algo": round(traffic / info["algo_bytes_per_launch"], 3),
               "commands": cmds}
        with open(os.path.join(ROOT, "profiles", f"{stage}_hbm_traffic.json"), "w") as fh:
            json.dump(rec, fh, indent=1)
        out[stage] = rec
    return out


def mfma_record(csv_path, bench_json, cmds):
    """Turns one rocprofv3 --pmc pass (SQ_VALU_MFMA_BUSY_CYCLES, SQ_BUSY_CYCLES,
    GRBM_GUI_ACTIVE) over bench.py into profiles/mfma_busy.json.  Per stage, over the timed
    region's launches (the last ones of the stage's kernels in the run): SQ_VALU_MFMA_BUSY_CYCLES
    sums the matrix units' busy cycles over the 1024 SIMDs (a 32x32x16 bf16 MFMA keeps one busy
    for 32 cycles, so it counts 1/1024 of the MFMA FLOPs); GRBM_GUI_ACTIVE sums the active cycles
    of the 8 XCDs.  mfma_busy_frac = busy / (GRBM_GUI_ACTIVE / 8 x 1024): the share of the
    launch the matrix units are busy at the clock they ran at; clock_ghz = (GRBM_GUI_ACTIVE / 8)
    / duration; mfma_tflops = the MFMA FLOPs issued per second."""
    import csv
    import hashlib
    with open(bench_json) as fh:
        bench = [json.loads(ln) for ln in fh if ln.startswith("{")][-1]
    with open(csv_path) as fh:
        rows = list(csv.DictReader(fh))
    by = {}
    for r in rows:
        d = by.setdefault(int(r["Dispatch_Id"]), {"name": r["Kernel_Name"],
                                                    "ns": int(r["End_Timestamp"]) -
                                                    int(r["Start_Timestamp"])})
        d[r["Counter_Name"]] = float(r["Counter_Value"])
    order = sorted(by)
    xcd, simds = 8, 1024
    out = {"commands": cmds,
           "formula": {"mfma_busy_frac": "SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / 8 * 1024)",
                       "clock_ghz": "(GRBM_GUI_ACTIVE / 8) / duration",
                       "mfma_tflops": "SQ_VALU_MFMA_BUSY_CYCLES * 1024 / duration (32768 FLOP "
                                      "per 32 busy cycles of a 32x32x16 bf16 MFMA)"},
           "stages": {}}
    for stage, info in bench["stages"].items():
        keys = STAGE_KERNEL.get(stage, ())
        ds = [d for d in order if any(k in by[d]["name"] for k in keys)][-info["launches"]:]
        if not ds:
            continue
        tot = {c: sum(by[d].get(c, 0.0) for d in ds) for c in
               ("SQ_VALU_MFMA_BUSY_CYCLES", "SQ_BUSY_CYCLES", "GRBM_GUI_ACTIVE")}
        ns = sum(by[d]["ns"] for d in ds)
        busy, act = tot["SQ_VALU_MFMA_BUSY_CYCLES"], tot["GRBM_GUI_ACTIVE"] / xcd
        src = os.path.join("paper_2506_14107_amd", "csrc", KERNEL_SOURCE[stage])
        out["stages"][stage] = {
            "kernel": by[ds[0]]["name"], "launches": len(ds), "counters": tot,
            "avg_launch_us": round(ns / len(ds) / 1e3, 2),
            "source": src,
            "source_sha256": hashlib.sha256(open(os.path.join(ROOT, src), "rb").read()).hexdigest(),
            "clock_ghz": round(act / ns, 3) if ns else None,
            "mfma_busy_frac": round(busy / max(act * simds, 1.0), 4),
            "mfma_tflops": round(busy * 1024 / ns * 1e-3, 1) if ns else None}
    with open(os.path.join(ROOT, "profiles", "mfma_busy.json"), "w") as fh:
        json.dump(out, fh, indent=1)
    return out


def calibrate(enc, x, G, target, iters=24, lo=-1.0, hi=1.0):
    """Bisection of tau in [lo, hi] so that the batch's reuse rate is within 0.01 of target
    (the cosine gate's tau lies in [-1, 1]; the decision MLP's threshold on d is wider)."""
    import torch
    # reuse(lo) high, reuse(hi) low
    best = None
    for _ in range(iters):
        mid = 0.5 * (lo + hi)
        _, mk, _ = enc.encode(x, G, mid)
        torch.cuda.synchronize()
        rho = reuse_of(mk.cpu().numpy(), G)
        if best is None or abs(rho - target) < abs(best[1] - target):
            best = (mid, rho)
        if abs(rho - target) <= 0.01:
            break
        if rho > target:
            lo = mid
        else:
            hi = mid
    return best


def cpu_baseline(w, blob, frames, taus, groups_per_level=2):
    """The CPU oracle on whole groups of the same frames: fp64 at each level's threshold
    (`groups_per_level` groups per level), its fp32 variant (one group at the last level) and
    reuse off (tau = -inf, fp64, one group)."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([t.get("num_threads", 1) for t in threadpool_info()] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    G = w.group_size
    ngroups = frames.shape[0] // G

    def run(levels, per, dtype):
        done, t0 = 0, time.time()
        for k, tau in enumerate(levels):
            for gsel in range(per):
                g0 = ((k * per + gsel) * 5 % ngroups) * G   # groups spread over the input
                oracle.encode(frames[g0:g0 + G], blob, w.model.as_dict(), G, tau=tau, dtype=dtype)
                done += G
        dt = time.time() - t0
        return done, dt

    n64, t64 = run(taus, groups_per_level, np.float64)
    n32, t32 = run(taus[-1:], 1, np.float32)
    nd, td = run([float("-inf")], 1, np.float64)
    return {"value": round(n64 / t64, 3), "unit": "frames/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{n64} frames ({n64 // G} groups of {G}: {groups_per_level} per reuse level "
                      f"at the bench's thresholds), fp64 NumPy, {t64:.1f} s",
            "fp32": {"value": round(n32 / t32, 3), "unit": "frames/s",
                     "sample": f"{n32} frames (one group at the last reuse level), the oracle "
                               f"in fp32, {t32:.1f} s"},
            "dense": {"value": round(nd / td, 3), "unit": "frames/s",
                      "sample": f"{nd} frames (one group) with reuse off (tau = -inf), fp64, "
                                f"{td:.1f} s"}}


def measured_peaks():
    """What this chip sustains, beside its nominal peaks: the library's MFMA-loop probe (four
    independent v_mfma_f32_32x32x16_bf16 chains of random register operands per wavefront, two
    blocks of four wavefronts per CU, all resident at once, no memory traffic) and a 1 GiB
    device-to-device copy (bytes read + written), best of three timed launches each, outside
    the timed region."""
    import torch
    from paper_2506_14107_amd.dejavu import dv_mfma_probe
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    blocks = 2 * cus
    sink = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    cur = torch.cuda.current_stream()

    def best(fn, work):
        fn()
        torch.cuda.synchronize()
        rates = []
        for _ in range(3):
            s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            s.record()
            fn()
            e.record()
            torch.cuda.synchronize()
            rates.append(work / (s.elapsed_time(e) * 1e-3))
        return max(rates)

    iters = 40000
    flops = dv_mfma_probe(blocks, iters, sink.data_ptr(), cur.cuda_stream)
    mfma = best(lambda: dv_mfma_probe(blocks, iters, sink.data_ptr(), cur.cuda_stream), flops)
    src = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    copy = best(lambda: dst.copy_(src), 2.0 * src.numel() * 4)
    del src, dst, sink
    return {"mfma_bf16_tflops": round(mfma / 1e12, 1), "hbm_copy_gbs": round(copy / 1e9, 1),
            "how": f"MFMA-loop probe ({blocks} blocks x 4 wavefronts x {iters} rounds of 4 "
                   "independent 32x32x16 bf16 chains of random operands) and a 1 GiB device copy, best of 3"}


def operating_points(name):
    """Thresholds of the workload's reuse levels from the fixture the parity tests use
    (calibrated with the CPU oracle by tests/golden/make_operating_points.py), or None."""
    path = os.path.join(ROOT, "tests", "golden", "operating_points.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        ops = json.load(fh)["workloads"].get(name)
    return {lv["target"]: lv["tau"] for lv in ops["levels"]} if ops else None


def render(video, S, n, workers=8):
    """Frames 0 .. n-1 of a recipe, rendered in parallel chunks (each frame depends only on the
    recipe and its index)."""
    if n <= 256:
        return synth.render_frames(video, S, 0, n)
    from concurrent.futures import ProcessPoolExecutor
    chunk = (n + workers - 1) // workers
    starts = list(range(0, n, chunk))
    out = np.empty((n, 3, S, S), np.float32)
    with ProcessPoolExecutor(workers) as ex:
        for s0, fr in zip(starts, ex.map(synth.render_frames, [video] * len(starts),
                                         [S] * len(starts), starts,
                                         [min(chunk, n - s0) for s0 in starts])):
            out[s0:s0 + fr.shape[0]] = fr
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="vit_l14")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--frames", type=int, default=0,
                    help="frames per encode (default: the workload's whole clip; the handle "
                         "keeps the workload's batch size)")
    ap.add_argument("--calibrate", action="store_true",
                    help="bisect each level's threshold on the GPU instead of taking the "
                         "oracle-calibrated operating points (always done with --restore, "
                         "--decision, --reorder)")
    ap.add_argument("--restore", action="store_true",
                    help="with the restoration layer on reused tokens (random restoration weights)")
    ap.add_argument("--decision", action="store_true",
                    help="gate with the learned decision MLP (random decision weights; the "
                         "threshold on its output is calibrated like tau)")
    ap.add_argument("--reorder", action="store_true",
                    help="reordered I/P/B referencing with past and future references")
    ap.add_argument("--streams", type=int, default=1,
                    help="with --stream-chunk: this many independent streams, one handle and one "
                         "HIP stream each, every one encoding the whole batch; calls are issued "
                         "round-robin (frames/s count all streams' frames; no roofline)")
    ap.add_argument("--stream-chunk", type=int, default=0,
                    help="deliver each batch to the timed encodes as a stream of calls of this "
                         "many frames (dv_stream_encode; groups span calls; a reordered stream "
                         "is flushed at the end)")
    ap.add_argument("--split", type=int, default=1,
                    help="encode the clip as this many contiguous parts of whole groups at the "
                         "same time, one handle (batches of 1/K of the workload's) and one HIP "
                         "stream each; bit-identical results; no roofline (the parts' kernels "
                         "share the chip, so no launch's duration is its own)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one plain 1 GiB device-to-device copy (HBM counter calibration)")
    ap.add_argument("--traffic-record", nargs=3, metavar=("FETCH_CSV", "WRITE_CSV", "BENCH_OUT"),
                    help="write profiles/<stage>_hbm_traffic.json from two rocprofv3 --pmc passes "
                         "(FETCH_SIZE, WRITE_SIZE) over bench.py --copy-calibration and that "
                         "run's output line; no GPU work")
    ap.add_argument("--mfma-record", nargs=2, metavar=("PMC_CSV", "BENCH_OUT"),
                    help="write profiles/mfma_busy.json from a rocprofv3 --pmc pass "
                         "(SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CYCLES GRBM_GUI_ACTIVE) over bench.py "
                         "and that run's output line; no GPU work")
    ap.add_argument("--command", action="append", default=[],
                    help="with --traffic-record: the profiling commands, kept in the record")
    args = ap.parse_args()
    if args.mfma_record:
        rec = mfma_record(*args.mfma_record, args.command)
        for st, r in rec["stages"].items():
            print(f"{st}: MFMA busy {r['mfma_busy_frac']} at {r['clock_ghz']} GHz, "
                  f"{r['mfma_tflops']} TFLOP/s issued, {r['avg_launch_us']} us per launch")
        return
    if args.traffic_record:
        recs = traffic_record(*args.traffic_record, args.command)
        for st, r in recs.items():
            print(f"{st}: {r['traffic_bytes_per_launch'] / 1e6:.1f} MB per launch, "
                  f"{r['traffic_over_algo']}x algorithmic")
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU: --gpus {args.gpus} is not supported (this path runs "
              "on a single MI355X; groups are independent, see the sharding notes)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2506_14107_amd.dejavu import Encoder, dv_workspace_bytes

    w = synth.get_config(args.workload)
    m = w.model
    if args.restore:
        import dataclasses
        m = dataclasses.replace(m, restore=True)
        w = dataclasses.replace(w, model=m)
    if args.decision:
        import dataclasses
        m = dataclasses.replace(m, decision=True)
        w = dataclasses.replace(w, model=m)
    if args.reorder:
        import dataclasses
        m = dataclasses.replace(m, reorder=True)
        w = dataclasses.replace(w, model=m)
    G, B = w.group_size, w.batch_frames
    F = args.frames or w.n_frames           # frames per encode
    batches = -(-F // ((B // G) * G))        # internal batches per encode
    t0 = time.time()
    blob = synth.make_blob(m, w.weight_seed)
    frames = render(w.video, m.image_size, F)
    log(f"[bench] {w.name}: {F} frames in {batches} batches of <= {B}, inputs ready in "
        f"{time.time() - t0:.1f} s")
    enc = Encoder(m, blob, B)
    x = torch.from_numpy(frames).cuda()
    targets = w.reuse_targets or (None,)
    ops = None if (args.calibrate or m.restore or m.decision or m.reorder) else \
        operating_points(w.name)
    taus = []
    for tgt in targets:
        if tgt is None:
            tau, how = float(np.float32(w.tau)), "fixed"
        elif ops is not None:
            tau, how = ops[tgt], "operating point"
        else:
            bracket = {"lo": -16.0, "hi": 16.0} if m.decision else {}
            tau, _ = calibrate(enc, x[:B], G, tgt, **bracket)
            how = "GPU bisection on the first batch"
        taus.append(float(np.float32(tau)))
        log(f"[bench] target reuse {tgt}: tau {tau!r} ({how})")

    # per-level reuse maps and active rows (deterministic: same as in the timed region), and the
    # embeddings' cosine to those of the same kernels with reuse off (the paper's accuracy proxy)
    e_dense, _, _ = enc.encode(x, G, float("-inf"), want_masks=False)
    levels = []
    for tau in taus:
        e, mk, _ = enc.encode(x, G, tau)
        torch.cuda.synchronize()
        mk = mk.cpu().numpy()
        cos = torch.nn.functional.cosine_similarity(e.double(), e_dense.double(), dim=1)
        cos = cos.cpu().numpy()[[f for f in range(F) if f % G]]
        levels.append({"tau": tau, "reuse": reuse_of(mk, G), "Ml": active_rows(mk, G),
                       "cos": (float(cos.mean()), float(cos.min()))})

    # the dominant stage: one profiled pass over every level (stage times also logged per level)
    prof = {}
    for lv in levels + [{"tau": float("-inf"), "reuse": 0.0}]:
        enc.profile(True)
        enc.encode(x, G, lv["tau"], want_masks=False)
        torch.cuda.synchronize()
        p = enc.profile_read()
        enc.profile(False)
        log(f"[bench] stage ms at reuse {lv['reuse']:.2f} (tau {lv['tau']:.4f}): "
            + ", ".join(f"{k} {v[0]:.2f}" for k, v in p.items() if v[1]))
        if lv["tau"] != float("-inf"):
            for k, v in p.items():
                a = prof.get(k, (0.0, 0))
                prof[k] = (a[0] + v[0], a[1] + v[1])
    dominant = max(prof, key=lambda s: prof[s][0])
    log("[bench] stage ms per sweep: " + ", ".join(f"{k} {v[0]:.2f}" for k, v in prof.items() if v[1]))

    S = max(1, args.streams) if args.stream_chunk else 1
    if S > 1:   # small handles: one call's frames plus a group of carried-over frames
        encs = [Encoder(m, blob, min(F, args.stream_chunk + G)) for _ in range(S)]
        hs = [torch.cuda.Stream() for _ in range(S)]
    K = max(1, args.split)
    if K > 1:   # contiguous parts of whole groups, one handle and HIP stream each
        if args.stream_chunk or F % (K * G):
            raise SystemExit("--split needs whole calls and a frame count that splits into "
                             f"{K} parts of whole groups of {G}")
        part = F // K
        part_cap = min(part, max(G, (B // K) // G * G))
        kencs = [Encoder(m, blob, part_cap) for _ in range(K)]
        khs = [torch.cuda.Stream() for _ in range(K)]

    def encode_all(tau):
        """One encode of the batch: one call, or a stream of calls of --stream-chunk frames (of
        --streams concurrent streams)."""
        if S > 1:
            cur = torch.cuda.current_stream()
            for e, st in zip(encs, hs):
                st.wait_stream(cur)
                e.stream_reset()
            for k in range(0, F, args.stream_chunk):
                for e, st in zip(encs, hs):
                    with torch.cuda.stream(st):
                        e.stream_encode(x[k:k + args.stream_chunk], G, tau, want_masks=False,
                                        stream=st)
            for e, st in zip(encs, hs):
                with torch.cuda.stream(st):
                    e.stream_flush(want_masks=False, stream=st)
                cur.wait_stream(st)
            return
        if K > 1:
            cur = torch.cuda.current_stream()
            for k, (e, st) in enumerate(zip(kencs, khs)):
                st.wait_stream(cur)
                with torch.cuda.stream(st):
                    e.encode(x[k * part:(k + 1) * part], G, tau, want_masks=False, stream=st)
            for st in khs:
                cur.wait_stream(st)
            return
        if not args.stream_chunk:
            enc.encode(x, G, tau, want_masks=False)
            return
        enc.stream_reset()
        for k in range(0, F, args.stream_chunk):
            enc.stream_encode(x[k:k + args.stream_chunk], G, tau, want_masks=False)
        enc.stream_flush(want_masks=False)   # frames held by a reordered stream

    # dense reference (same kernels, reuse off)
    def time_calls(tau_list, steps, warmup, profile_stage=None):
        for _ in range(warmup):
            for tau in tau_list:
                encode_all(tau)
        torch.cuda.synchronize()
        if profile_stage:
            enc.profile([profile_stage])
        # an event after every step: the whole region's time and each step's
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        evs[0].record()
        for k in range(steps):
            for tau in tau_list:
                encode_all(tau)
            evs[k + 1].record()
        torch.cuda.synchronize()
        ms = evs[0].elapsed_time(evs[-1])
        per_step = [evs[k].elapsed_time(evs[k + 1]) for k in range(steps)]
        st = None
        if profile_stage:
            st = enc.profile_read()[profile_stage]
            enc.profile(False)
        return ms, st, per_step

    per_level = []
    for lv in levels:
        ms, _, _ = time_calls([lv["tau"]], max(2, args.steps), 1)
        per_level.append(S * F * max(2, args.steps) / ms * 1e3)
    dense_ms, _, _ = time_calls([float("-inf")], max(2, args.steps), 1)
    dense_fps = S * F * max(2, args.steps) / dense_ms * 1e3

    # the timed region: K steps of the whole sweep, dominant stage timed with HIP events
    total_ms, st, step_ms = time_calls(taus, args.steps, args.warmup,
                                       profile_stage=dominant if S == 1 and K == 1 else None)
    frames_done = S * F * len(taus) * args.steps
    value = frames_done / total_ms * 1e3

    peaks = measured_peaks()
    log(f"[bench] measured peaks: {peaks['mfma_bf16_tflops']} TFLOP/s bf16 MFMA loop, "
        f"{peaks['hbm_copy_gbs']} GB/s device copy")

    # roofline of the dominant kernel
    flops = args.steps * sum(stage_flops(dominant, m, Ml) for lv in levels for Ml in lv["Ml"])
    stage_ms, launches = st if st is not None else (0.0, 0)
    if S > 1 or K > 1:   # concurrent streams: no single kernel's launches to time
        roof = None
    elif flops > 0:
        achieved = flops / (stage_ms * 1e-3) / 1e12
        peak = PEAK_BF16_TFLOPS if m.dtype == "bf16" else PEAK_FP32_TFLOPS
        algo_b = args.steps * sum(stage_bytes(dominant, m, Ml) for lv in levels for Ml in lv["Ml"])
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4),
                "traffic": measured_traffic(dominant, w.name == "vit_l14" and not (
                    args.frames or args.restore or args.decision or args.reorder
                    or args.stream_chunk)),
                "measured_peak": peaks["mfma_bf16_tflops"] if m.dtype == "bf16" else None,
                "frac_of_measured_peak": round(achieved / peaks["mfma_bf16_tflops"], 4)
                if m.dtype == "bf16" else None,
                "kernel": dominant, "launches": launches,
                "avg_launch_us": round(stage_ms / max(launches, 1) * 1e3, 2),
                "algo_flops_per_launch": round(flops / max(launches, 1)),
                "algo_bytes_per_launch": round(algo_b / max(launches, 1))}
    else:
        roof = {"bound": "hbm", "achieved": None, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": None, "traffic": None, "kernel": dominant, "launches": launches}

    # FLOPs of the whole sweep vs dense, for the ideal (skipped-FLOP) speedup
    D, N, P = m.width, m.n_tokens, m.n_patches
    per_row = 24.0 * D * D + 4.0 * N * D
    patch = 2.0 * P * 3 * m.patch * m.patch * D * F
    sweep = []
    for lv, fps in zip(levels, per_level):
        algo = patch + per_row * float(np.sum(lv["Ml"]))
        dense = patch + per_row * F * N * m.depth
        sweep.append({"tau": lv["tau"], "reuse": round(lv["reuse"], 4),
                      "frames_per_s": round(fps, 1), "speedup_vs_dense": round(fps / dense_fps, 3),
                      "ideal_speedup": round(dense / algo, 3),
                      "emb_cos_vs_dense_mean": round(lv["cos"][0], 5),
                      "emb_cos_vs_dense_min": round(lv["cos"][1], 5)})

    if args.copy_calibration:   # one plain copy kernel of known size for the HBM counters
        src = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log("[bench] copy calibration: 1 GiB device-to-device copy done")
        del src, dst

    # per stage: launches and algorithmic bytes per launch in the timed region, and from the
    # profiled pass over the sweep (one encode per level, HIP events around every launch) the
    # time per sweep and the achieved fractions of the MFMA and HBM peaks
    launches_per_stage = args.steps * len(levels) * m.depth * batches
    peak_f = PEAK_BF16_TFLOPS if m.dtype == "bf16" else PEAK_FP32_TFLOPS
    stages = {}

    def account(stg, flops_sweep, bytes_sweep, launches):
        ms = prof.get(stg, (0.0, 0))[0]
        rec = {"launches": launches, "algo_bytes_per_launch":
               round(bytes_sweep * args.steps / launches) if launches else 0,
               "ms_per_sweep": round(ms, 3)}
        if ms > 0:
            if flops_sweep:
                rec["tflops"] = round(flops_sweep / ms * 1e-9, 1)
                rec["mfma_frac"] = round(flops_sweep / ms * 1e-9 / peak_f, 4)
            rec["gbs"] = round(bytes_sweep / ms * 1e-6, 1)
            rec["hbm_frac"] = round(bytes_sweep / ms * 1e-6 / PEAK_HBM_GBS, 4)
        stages[stg] = rec

    for stg in ("qkv", "oproj", "fc1", "fc2", "attn"):
        fl = sum(stage_flops(stg, m, Ml) for lv in levels for Ml in lv["Ml"])
        by = sum((attn_bytes(m, Ml, F) if stg == "attn" else stage_bytes(stg, m, Ml))
                 for lv in levels for Ml in lv["Ml"])
        account(stg, fl, by, launches_per_stage)
    for stg in ("gate", "ln2", "compact"):
        by = sum(row_stage_bytes(stg, m, (lv["Ml"][l - 1] if l else F * N), lv["Ml"][l], F)
                 for lv in levels for l in range(m.depth))
        account(stg, 0.0, by, launches_per_stage)
    img = 3 * m.image_size * m.image_size
    account("patch", 2.0 * P * 3 * m.patch * m.patch * D * F * len(levels),
            (F * img * 4 + F * N * D * 4) * len(levels), args.steps * len(levels) * batches)

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(w, blob, frames, taus)

    out = {
        "metric": METRIC if w.name == "vit_l14" else
                  f"frames/s {w.name} at " + "/".join(f"{t:.0%}" for t in targets if t is not None)
                  + " reuse; packed-GEMM MFMA util; speedup vs dense",
        "value": round(value, 2), "unit": "frames/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(total_ms / args.steps, 3),
        "step_ms": {"median": round(float(np.median(step_ms)), 3),
                    "min": round(min(step_ms), 3), "max": round(max(step_ms), 3)},
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if m.dtype == "bf16" else "f32", "data": "synthetic",
        "config": {"workload": f"{w.name}: {m.image_size}px patch {m.patch} ({N} tokens), depth "
                               f"{m.depth}, width {D}, {m.heads} heads, MLP {m.mlp}; {F} frames "
                               f"per encode in batches of {B}, groups of {G}; "
                               + ("restoration MLP (hidden 128) on reused tokens; " if m.restore
                                  else "")
                               + ("learned decision MLP gate (hidden 64); " if m.decision
                                  else "")
                               + ("reordered I/P/B referencing (past and future anchors); "
                                  if m.reorder else "")
                               + (f"streamed in calls of {args.stream_chunk} frames; "
                                  if args.stream_chunk else "")
                               + (f"{S} concurrent streams (one handle and HIP stream each, "
                                  f"each encoding the batch); " if S > 1 else "")
                               + (f"split into {K} concurrent parts of {part} frames (one "
                                  f"handle, batches of {part_cap}, and one HIP stream each); "
                                  if K > 1 else "")
                               + "reuse levels "
                               + "/".join(f"{t:.0%}" for t in targets if t is not None),
                   "frames_per_step": S * F * len(taus), "group_size": G},
        "sweep": sweep,
        "dense_frames_per_s": round(dense_fps, 1),
        "roofline": roof,
        "stages": stages,
        "cpu_baseline": cpu,
        "measured_peaks": peaks,
        "workspace_bytes": dv_workspace_bytes(enc.handle),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
