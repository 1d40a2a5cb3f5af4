"""Reordered I/P/B referencing with past and future references (Section 3.1) through the C ABI
against the CPU oracle.  Decisions and sources are teacher-forced: the oracle replays the GPU's
map (1 = reused from the past reference, 2 = from the future one) and judges each choice by its
own cosines outside a 1e-3 band; outputs meet the usual bar.  A B frame equal to its future
anchor copies it bitwise; internal batching (with its look-ahead I frame) and reuse off are
bitwise properties."""
import dataclasses

import numpy as np
import pytest

import oracle
import synth
from synth.configs import ModelConfig

from .gpu_util import check_close, dev, encoder, host, require_gpu
from .test_gpu_decision import decision_band
from .test_gpu_parity import _video

pytestmark = pytest.mark.gpu

TINY = synth.get_config("tiny")
TINY_O = dataclasses.replace(TINY.model, reorder=True)
SMALL_O = ModelConfig(64, 16, 2, 128, 2, 256, "bf16", reorder=True)
MID_O = ModelConfig(112, 16, 3, 256, 4, 512, "bf16", reorder=True)
N257_O = ModelConfig(224, 14, 2, 128, 2, 256, "bf16", reorder=True)
DH80_O = ModelConfig(112, 16, 2, 640, 8, 1280, "bf16", reorder=True)
MID_OD = ModelConfig(112, 16, 3, 256, 4, 512, "bf16", decision=True, reorder=True)

BAND = 1e-3


def reorder_parity(mg, r, tau=None):
    """(decisions off, sources off, fraction inside the band): outside a 1e-3 band the GPU's
    decision is [s >= tau] (when tau is given) and a reused token's source is the reference
    with the larger cosine (2 = the future one)."""
    s, cp, cf = r["cos"], r["cos_past"], r["cos_fut"]
    ev = ~np.isnan(s)
    reuse = mg != 0
    bad = 0
    inside = 0.0
    if tau is not None:
        ok = ev & (np.abs(s - tau) >= BAND)
        bad = int(np.sum(reuse[ok] != (s[ok] >= tau)))
        inside = float(np.mean(~ok[ev])) if ev.any() else 0.0
    two = ev & reuse & ~np.isnan(cf) & (np.abs(cf - cp) >= BAND)
    bad_src = int(np.sum((mg[two] == 2) != (cf[two] > cp[two])))
    return bad, bad_src, inside


def _run(m, blob, fr, G, tau=None, batch=16, masks=None):
    torch = require_gpu()
    enc = encoder(m, blob, batch)
    if masks is None:
        emb, mk, toks = enc.encode(dev(fr), G, float(tau), want_tokens=True)
    else:
        emb, mk, toks = enc.encode_masked(dev(fr), G, dev(masks), want_tokens=True)
    torch.cuda.synchronize()
    return host(emb), host(mk), host(toks)


def _frames(m, F, seed):
    if m.dtype == "f32":
        return synth.render_frames(TINY.video, m.image_size, 0, F)
    return _video(m, F, seed=seed, sigma=0.02, pan=1.0)


@pytest.mark.parametrize("m,G,F,batch", [(TINY_O, 4, 8, 8), (SMALL_O, 8, 16, 16),
                                         (MID_O, 8, 21, 8), (N257_O, 8, 16, 16),
                                         (DH80_O, 4, 10, 8), (SMALL_O, 12, 30, 16)],
                         ids=["tiny", "small", "mid-batched", "n257", "dh80-batched",
                              "p-chain-g12"])
def test_reorder_gate_parity(m, G, F, batch):
    blob = synth.make_blob(m, 51, perturb_ln=True)
    fr = _frames(m, F, 51)
    dt = "f32" if m.dtype == "f32" else "bf16"
    futures = 0
    for tau in ((0.95,) if m.dtype == "f32" else (0.6, 0.9, 0.99)):
        tau = float(np.float32(tau))
        emb, mg, toks = _run(m, blob, fr, G, tau, batch)
        r = oracle.encode(fr, blob, m.as_dict(), G, masks=(mg != 0), sources=(mg == 2))
        bad, bad_src, inside = reorder_parity(mg, r, tau)
        assert bad == 0 and bad_src == 0, \
            f"tau={tau}: {bad} decisions and {bad_src} sources off ({inside:.2%} inside the band)"
        assert not mg[::G].any() and not mg[:, :, 0].any()
        check_close(emb, r["emb"], dt, f"embeddings tau={tau}")
        check_close(toks, r["tokens"], dt, f"tokens tau={tau}")
        futures += int((mg == 2).sum())
    assert futures > 0, "no token was reused from a future reference"


@pytest.mark.parametrize("m", [SMALL_O, MID_O], ids=["small", "mid"])
def test_reorder_future_copy_is_bitwise(m):
    """Frame 2 (B_dist2 between anchors 0 and 4) equal to its future anchor: every token reused
    from frame 4 at layer 0, and frame 2's outputs are frame 4's, bit for bit."""
    blob = synth.make_blob(m, 52)
    fr = _video(m, 9, seed=52, sigma=0.02)
    fr[4] = np.random.default_rng(53).standard_normal(fr[4].shape).astype(np.float32)
    fr[2] = fr[4]
    emb, mg, toks = _run(m, blob, fr, 8, 0.9)
    assert (mg[2, 0, 1:] == 2).all() and (mg[2, :, 1:] != 0).all()
    assert np.array_equal(toks[2], toks[4]) and np.array_equal(emb[2], emb[4])


def test_reorder_batching_is_bitwise():
    m = SMALL_O
    blob = synth.make_blob(m, 54)
    fr = _frames(m, 27, 54)   # three full groups and a short one
    outs = [_run(m, blob, fr, 8, 0.9, batch) for batch in (8, 16, 32)]
    for o in outs[1:]:
        for a, b, what in zip(o, outs[0], ("embeddings", "masks", "tokens")):
            assert np.array_equal(a, b), f"{what} depend on the batch size"


@pytest.mark.parametrize("m", [TINY_O, MID_O], ids=["tiny", "mid"])
def test_reorder_off_equivalences_are_bitwise(m):
    blob = synth.make_blob(m, 55)
    fr = _frames(m, 12, 55)
    base = dataclasses.replace(m, reorder=False)
    dense = _run(base, blob, fr, 4, -np.inf)
    for mm, tau in ((m, -np.inf), (m, 2.0)):   # reuse off; the gate on, reusing nothing
        got = _run(mm, blob, fr, 4, tau)
        assert not got[1].any()
        for a, b, what in zip(got, dense, ("embeddings", "masks", "tokens")):
            assert np.array_equal(a, b), f"{what} differ (tau={tau})"


@pytest.mark.parametrize("m,G", [(SMALL_O, 4), (MID_O, 8)], ids=["small", "mid"])
def test_reorder_injection(m, G):
    blob = synth.make_blob(m, 56, perturb_ln=True)
    F = 13
    fr = _frames(m, F, 56)
    mk = (np.random.default_rng(57).random((F, m.depth, m.n_tokens)) < 0.6).astype(np.uint8)
    emb, eff, toks = _run(m, blob, fr, G, masks=mk, batch=8)
    assert np.array_equal(eff != 0, oracle.encode(fr, blob, m.as_dict(), G, masks=mk)["masks"] != 0)
    r = oracle.encode(fr, blob, m.as_dict(), G, masks=mk, sources=(eff == 2))
    _, bad_src, _ = reorder_parity(eff, r)
    assert bad_src == 0, f"{bad_src} sources differ outside the band"
    check_close(emb, r["emb"], "bf16", "embeddings")
    check_close(toks, r["tokens"], "bf16", "tokens")


def test_reorder_with_decision_mlp():
    m = MID_OD
    w = synth.make_weights(m, 58, perturb_ln=True)
    blob = synth.pack_weights(w, m)
    G, F = 8, 16
    fr = _frames(m, F, 58)
    r0 = oracle.encode(fr, blob, m.as_dict(), G, tau=0.0)
    tau = float(np.float32(np.quantile(r0["dec"][~np.isnan(r0["dec"])], 0.4)))
    emb, mg, toks = _run(m, blob, fr, G, tau)
    r = oracle.encode(fr, blob, m.as_dict(), G, masks=(mg != 0), sources=(mg == 2))
    d = r["dec"]
    ev = ~np.isnan(d)
    ok = ev & (np.abs(d - tau) >= decision_band(w, m, r["t"]))
    assert int(np.sum((mg[ok] != 0) != (d[ok] > tau))) == 0
    _, bad_src, _ = reorder_parity(mg, r)
    assert bad_src == 0
    assert 0.1 < oracle.reuse_rate(mg, G) < 0.95
    check_close(emb, r["emb"], "bf16", "embeddings")
    check_close(toks, r["tokens"], "bf16", "tokens")


def test_reorder_needs_group_multiple_of_4():
    from paper_2506_14107_amd import dejavu as dj
    m = SMALL_O
    blob = synth.make_blob(m, 59)
    fr = _frames(m, 6, 59)
    enc = encoder(m, blob, 8)
    with pytest.raises(dj.DejaVuError) as e:
        enc.encode(dev(fr), 6, 0.9)
    assert e.value.code == dj.DV_EINVAL and "multiple of 4" in dj.dv_last_error()
    # with restoration, chains of sources are bounded: at most 60 frames per group
    mr = dataclasses.replace(m, restore=True)
    enc = encoder(mr, synth.make_blob(mr, 59), 64)
    with pytest.raises(dj.DejaVuError) as e:
        enc.encode(dev(fr[:4]), 64, 0.9)
    assert e.value.code == dj.DV_EINVAL and "<= 60" in dj.dv_last_error()
    enc.encode(dev(fr[:4]), 60, 0.9)


TINY_OR = dataclasses.replace(TINY_O, restore=True)
MID_OR = ModelConfig(112, 16, 3, 256, 4, 512, "bf16", restore=True, reorder=True)


def longest_chain(mg, G):
    """Longest chain of reused sources in a map (out_masks codes: 1 past, 2 future)."""
    from oracle.reusevit import reference_frames
    F, L, N = mg.shape
    best = 0
    for l in range(L):
        for f in range(F):
            for i in range(N):
                g, n = f, 0
                while mg[g, l, i]:
                    n += 1
                    _, past, fut = reference_frames(g, G, F)
                    g = fut if mg[g, l, i] == 2 else past
                best = max(best, n)
    return best


@pytest.mark.parametrize("m,G,F,batch", [(TINY_OR, 4, 8, 8), (MID_OR, 8, 21, 8),
                                         (TINY_OR, 60, 61, 64)],
                         ids=["tiny", "mid-batched", "tiny-g60-longest-chains"])
def test_reorder_with_restoration(m, G, F, batch):
    """Restoration on reused rows under reordering: a reused row is its source's new row plus the
    restoration MLP of its input difference to the source, built along chains of sources."""
    w = synth.make_weights(m, 60, perturb_ln=True, std=0.05)
    blob = synth.pack_weights(w, m)
    fr = _frames(m, F, 60)
    dt = "f32" if m.dtype == "f32" else "bf16"
    for tau in ((0.95,) if m.dtype == "f32" else (0.9, 0.6)):
        tau = float(np.float32(tau))
        emb, mg, toks = _run(m, blob, fr, G, tau, batch)
        r = oracle.encode(fr, blob, m.as_dict(), G, masks=(mg != 0), sources=(mg == 2))
        bad, bad_src, inside = reorder_parity(mg, r, tau)
        assert bad == 0 and bad_src == 0, f"tau={tau}: {bad} decisions, {bad_src} sources off"
        assert 0.05 < oracle.reuse_rate(mg, G) < 0.99
        check_close(emb, r["emb"], dt, f"embeddings tau={tau}")
        check_close(toks, r["tokens"], dt, f"tokens tau={tau}")
    # the restoration changes reused rows: without it the outputs differ
    base = dataclasses.replace(m, restore=False)
    r0 = oracle.encode(fr, synth.pack_weights(w, base), base.as_dict(), G, masks=(mg != 0),
                       sources=(mg == 2))
    assert np.max(np.abs(r0["tokens"] - r["tokens"])) > 1e-3
    if G == 60:
        assert longest_chain(mg, G) == 16, "want chains of the maximum length"
    # batching (with the look-ahead I frame) does not change results
    again = _run(m, blob, fr, G, tau, 2 * batch)
    for a, b in zip(again, (emb, mg, toks)):
        assert np.array_equal(a, b)


def test_full_method_decision_restoration_reordering():
    """The paper's full method on the GPU: the decision MLP gating with reordered references and
    the restoration layer on reused rows, against the oracle replaying the GPU's map and sources
    (decisions judged outside the weight-derived margin)."""
    m = ModelConfig(112, 16, 3, 256, 4, 512, "bf16", restore=True, decision=True, reorder=True)
    w = synth.make_weights(m, 61, perturb_ln=True, std=0.05)
    blob = synth.pack_weights(w, m)
    G, F = 8, 17
    fr = _frames(m, F, 61)
    r0 = oracle.encode(fr, blob, m.as_dict(), G, tau=0.0)
    tau = float(np.float32(np.quantile(r0["dec"][~np.isnan(r0["dec"])], 0.4)))
    emb, mg, toks = _run(m, blob, fr, G, tau, 8)
    r = oracle.encode(fr, blob, m.as_dict(), G, masks=(mg != 0), sources=(mg == 2))
    d = r["dec"]
    ok = ~np.isnan(d) & (np.abs(d - tau) >= decision_band(w, m, r["t"]))
    assert int(np.sum((mg[ok] != 0) != (d[ok] > tau))) == 0
    assert reorder_parity(mg, r)[1] == 0
    assert 0.1 < oracle.reuse_rate(mg, G) < 0.95
    check_close(emb, r["emb"], "bf16", "embeddings")
    check_close(toks, r["tokens"], "bf16", "tokens")
