"""The learned decision gate (Section 3.3, decision layer) through the C ABI against the CPU
oracle.  Decisions are teacher-forced: the oracle replays the GPU's maps and judges each
decision by its own d_i, outside a margin derived from the MLP's weights and the feature
errors; outputs meet the usual bar.  Special weights reduce the MLP to the cosine gate, to
full reuse and to none, and must reproduce the GPU's runs of those modes bitwise."""
import dataclasses

import numpy as np
import pytest

import oracle
import synth
from synth.configs import ModelConfig

from .gpu_util import check_close, dev, encoder, host, require_gpu
from .pins import linear_decision
from .test_gpu_parity import _video

pytestmark = pytest.mark.gpu

TINY = synth.get_config("tiny")
TINY_D = dataclasses.replace(TINY.model, decision=True)
SMALL_D = ModelConfig(64, 16, 2, 128, 2, 256, "bf16", decision=True)
MID_D = ModelConfig(112, 16, 3, 256, 4, 512, "bf16", decision=True)
N257_D = ModelConfig(224, 14, 2, 128, 2, 256, "bf16", decision=True)
MID_RD = ModelConfig(112, 16, 3, 256, 4, 512, "bf16", restore=True, decision=True)

GELU_SLOPE = 1.13   # max |GELU'(z)| over the reals (at z ~ 1.4)
# Largest fraction of decisions the margin may leave unjudged: a wider band would let most
# decisions pass unchecked (about 1 % lie inside at ViT-L/14).
BAND_MAX = 0.05


def feature_errors(m):
    """Assumed bounds on the GPU's feature errors against the fp64 oracle: cosine (absolute)
    and class-token attention weight (relative).  bf16 operands: 1e-3 (the cosine gate's
    band) and 0.2 % (bf16 rounding of Q and K moves a score by about 2^-9 of its size, and the
    scores here are O(0.1)); fp32: 1e-4 and 0.01 %."""
    return (1e-3, 2e-3) if m.dtype == "bf16" else (1e-4, 1e-4)


def decision_band(w, m, t):
    """Per-token margin on d_i inside which GPU and oracle may decide differently: the MLP's
    sensitivity to s and t (|GELU'| <= 1.13 through |w_2| |W_1|) times the feature errors."""
    es, et = feature_errors(m)
    band = np.zeros_like(t)
    for l in range(m.depth):
        W1, W2 = w[f"l{l}.W_d1"].astype(np.float64), w[f"l{l}.W_d2"][0].astype(np.float64)
        ks = GELU_SLOPE * np.sum(np.abs(W2) * np.abs(W1[:, 0]))
        kt = GELU_SLOPE * np.sum(np.abs(W2) * np.abs(W1[:, 1]))
        band[:, l] = ks * es + kt * (et * np.abs(t[:, l]) + 1e-6)
    return band


def decision_parity(mg, r, band, tau):
    """(mismatches outside the band, fraction of evaluated tokens inside it)."""
    d = r["dec"]
    ev = ~np.isnan(d)
    decided = ev & (np.abs(d - tau) >= band)
    bad = int(np.sum(mg.astype(bool)[decided] != (d[decided] > tau)))
    return bad, float(np.mean(~decided[ev]))


def _run(m, blob, fr, G, tau, batch=16):
    torch = require_gpu()
    emb, masks, toks = encoder(m, blob, batch).encode(dev(fr), G, float(tau), want_tokens=True)
    torch.cuda.synchronize()
    return host(emb), host(masks), host(toks)


def _case(m, seed, F=16):
    w = synth.make_weights(m, seed, perturb_ln=True)
    if m.dtype == "f32":
        fr = synth.render_frames(TINY.video, m.image_size, 0, F)
    else:
        fr = _video(m, F, seed=seed, sigma=0.02)
    return w, fr


def judged_thresholds(w, m, fr, G, blob, k=2, sep=0.15):
    """Operating points where the check has power: candidate thresholds at the 5 %, 10 %, ...,
    95 % quantiles of the oracle's decision values at the paper's tau = 0, each scored by the
    fraction of decisions inside the margin in the oracle's own run at that threshold; the k
    lowest-scoring candidates at least `sep` apart in quantile.  (Reused tokens carry an exact
    cosine of 1, so their d values cluster and a plain quartile can sit inside a cluster.)"""
    r0 = oracle.encode(fr, blob, m.as_dict(), G, tau=0.0)
    dv = r0["dec"][~np.isnan(r0["dec"])]
    scored = []
    for q in np.arange(0.05, 0.951, 0.05):
        tau = float(np.float32(np.quantile(dv, q)))
        r = oracle.encode(fr, blob, m.as_dict(), G, tau=tau)
        d, ev = r["dec"], ~np.isnan(r["dec"])
        inside = float(np.mean(np.abs(d[ev] - tau) < decision_band(w, m, r["t"])[ev]))
        scored.append((inside, q, tau))
    picked = []
    for inside, q, tau in sorted(scored):
        if all(abs(q - q2) >= sep for _, q2, _ in picked):
            picked.append((inside, q, tau))
        if len(picked) == k:
            break
    return [tau for _, _, tau in picked]


@pytest.mark.parametrize("m,G", [(TINY_D, 4), (SMALL_D, 8), (MID_D, 8), (N257_D, 8)],
                         ids=["tiny", "small", "mid", "n257"])
def test_decision_gate_parity(m, G):
    w, fr = _case(m, 41, F=8 if m is TINY_D else 16)
    blob = synth.pack_weights(w, m)
    # operating points: the paper's tau = 0 and two judged thresholds apart in the range
    checked = 0
    for tau in (0.0, *judged_thresholds(w, m, fr, G, blob)):
        tau = float(np.float32(tau))
        emb, mg, toks = _run(m, blob, fr, G, tau)
        r = oracle.encode(fr, blob, m.as_dict(), G, masks=mg)
        band = decision_band(w, m, r["t"])
        bad, inside = decision_parity(mg, r, band, tau)
        print(f"[decision {m.width}] tau {tau:.4f}: reuse {oracle.reuse_rate(mg, G):.3f}, "
              f"decisions off {bad}, in band {inside:.2%}", flush=True)
        assert bad == 0, f"tau={tau}: {bad} decisions differ outside the band ({inside:.1%} inside)"
        assert inside <= BAND_MAX, f"tau={tau}: band too wide to check ({inside:.1%} inside)"
        checked += 1
        dt = "f32" if m.dtype == "f32" else "bf16"
        check_close(emb, r["emb"], dt, f"embeddings tau={tau}")
        check_close(toks, r["tokens"], dt, f"tokens tau={tau}")
    assert checked == 3


@pytest.mark.parametrize("m,G,theta", [(TINY_D, 4, 0.95), (SMALL_D, 8, 0.9), (MID_D, 8, 0.75)],
                         ids=["tiny", "small", "mid"])
def test_decision_as_cosine_gate_is_bitwise(m, G, theta):
    """d = 5 (s - theta): the same maps and outputs as the cosine gate at tau = theta, although
    this path gates every token at every layer and copies reused rows."""
    w, fr = _case(m, 42, F=8 if m is TINY_D else 16)
    blob, th = linear_decision(w, m, 0, 5.0, theta)
    base = dataclasses.replace(m, decision=False)
    e0, k0, t0 = _run(base, synth.pack_weights(w, base), fr, G, th)
    e1, k1, t1 = _run(m, blob, fr, G, 0.0)
    assert 0.05 < k0.mean() < 0.95, "want a mixed map"
    assert np.array_equal(k0, k1), "maps differ"
    assert np.array_equal(e0, e1), "embeddings differ"
    assert np.array_equal(t0, t1), "tokens differ"


@pytest.mark.parametrize("m", [TINY_D, MID_D], ids=["tiny", "mid"])
def test_decision_full_none_and_tie_are_bitwise(m):
    """Frame-type weights: d = +0.5 reuses everything (== tau = +inf), d = -0.5 nothing
    (== tau = -inf), and d == 0 exactly recomputes (the tie of d > 0)."""
    w, fr = _case(m, 43, F=8)
    G = 4
    full = _run(m, synth.pack_weights(w, m), fr, G, np.inf)
    none = _run(m, synth.pack_weights(w, m), fr, G, -np.inf)
    for col, theta, want in ((3, 0.5, full), (2, 0.5, none), (3, 1.0, none)):
        blob, _ = linear_decision(w, m, col, 1.0, theta)
        got = _run(m, blob, fr, G, 0.0)
        for a, b, what in zip(got, want, ("embeddings", "masks", "tokens")):
            assert np.array_equal(a, b), f"{what} differ (type column {col}, theta {theta})"


@pytest.mark.parametrize("m", [SMALL_D, N257_D], ids=["small", "n257"])
def test_decision_attention_cue(m):
    """d = N (t - theta): nothing reused at layer 0 (t = 1/N there); at layer 1 the decisions
    follow the class-token attention weights of layer 0, computed by the GPU."""
    w, fr = _case(m, 44)
    G = 8
    N = m.n_tokens
    a, c = float(N), 10.0   # t scaled to O(1); GELU is the identity at z ~ 11 in fp32 too
    blob, th = linear_decision(w, m, 1, a, 1.01 / N, c)
    r0 = oracle.encode(fr, blob, m.as_dict(), G, tau=0.0)
    t1 = r0["t"][:, 1, 1:]
    theta = max(float(np.nanmedian(t1)), 1.01 / N)
    blob, th = linear_decision(w, m, 1, a, theta, c)
    emb, mg, toks = _run(m, blob, fr, G, 0.0)
    assert not mg[:, 0].any(), "t = 1/N at layer 0"
    assert 0.1 < mg[:, 1].mean() < 0.9, "want a mixed map at layer 1"
    r = oracle.encode(fr, blob, m.as_dict(), G, masks=mg)
    _, et = feature_errors(m)
    band = a * (et * np.abs(r["t"]) + 1e-6)
    bad, inside = decision_parity(mg, r, band, 0.0)
    print(f"[decision attention cue {m.n_tokens}] decisions off {bad}, in band {inside:.2%}",
          flush=True)
    assert bad == 0, f"{bad} decisions differ outside the band ({inside:.1%} inside)"
    assert inside <= BAND_MAX
    check_close(emb, r["emb"], "bf16", "embeddings")


def test_decision_with_restoration():
    m = MID_RD
    w, fr = _case(m, 45)
    blob = synth.pack_weights(w, m)
    G = 8
    tau = judged_thresholds(w, m, fr, G, blob, k=1)[0]
    emb, mg, toks = _run(m, blob, fr, G, tau)
    r = oracle.encode(fr, blob, m.as_dict(), G, masks=mg)
    bad, inside = decision_parity(mg, r, decision_band(w, m, r["t"]), tau)
    print(f"[decision with restoration] decisions off {bad}, in band {inside:.2%}", flush=True)
    assert bad == 0, f"{bad} decisions differ outside the band ({inside:.1%} inside)"
    assert inside <= BAND_MAX
    assert 0.1 < oracle.reuse_rate(mg, G) < 0.95
    check_close(emb, r["emb"], "bf16", "embeddings")
    check_close(toks, r["tokens"], "bf16", "tokens")
