"""Checks that pin the CPU oracle to things other than itself.

Each ``pin_*`` takes an oracle-like namespace (``encode``, ``cosine_rows``,
``gate_decision``, ``reuse_rate``) and raises AssertionError on failure.  The
oracle's own tests run them on ``oracle.reusevit``; the mutation test runs
them on copies of that module with a planted mistake and requires that at
least one pin fails for each mistake.

What pins what:
  library      dense forward == torch conv2d + TransformerEncoderLayer(norm_first) + layer_norm
  dense_vit    reuse off == the separately written dense ViT
  bruteforce   == the per-token loop implementation, gate and injection modes
  copy         tau=+inf: every non-reference frame is a bitwise copy of its reference
  ref_dense    reference frames equal the dense ViT for any tau; their mask rows are 0
  monotone     gate mode: a reused token stays reused in later layers
  static       identical frames are fully reused at layer 0 and copy the reference
  g1           group size 1 is the dense ViT
  groups       permuting whole groups permutes outputs; group-aligned splits change nothing
  inject_one   one injected reused token: its row copies the reference output and the other
               queries attend to the reference's K/V there (torch MHA with separate key input)
  extremes     tau=2 == reuse off, tau=-2 == tau=+inf
  star         every frame of a group references the group's first frame
  cosine       closed-form cosines; equal rows give exactly 1; tie cos == tau reuses
  partial      a short last group still has its first frame as reference
  rate         reuse-rate denominator: non-reference frames x N tokens x L layers
  restoration (the restoration MLP on reused rows, when the configuration enables it):
  restore_zero a zero output layer leaves every row and decision unchanged (bitwise)
  restore_brute == the per-token loop implementation, gate and injection modes
  restore_one  one injected reused token: reference output + the MLP (torch Linear/GELU) of its
               input difference; every other row as without restoration
  restore_static identical frames at tau=+inf: closed forms at layers 0 and 1
  decision layer (the learned gate, when the configuration enables it):
  decision_threshold an MLP that is a*(s - theta) gives the cosine gate's maps and outputs
  decision_attention  the class-token attention cue: 1/N before the first layer, then torch
               MultiheadAttention's head-averaged weights of the class query in the previous
               layer (also with a reference key/value substituted)
  decision_type      the frame-type cue is the P entry for every non-reference frame; a tie
               d == tau recomputes
  decision_mlp       the MLP itself == torch Linear/GELU/Linear on the features
  decision_brute     == the per-token loop implementation (with and without restoration)
  reordered referencing (I/P/B frames with past and future references):
  reorder_pattern    the reference graph of the paper's I -> (P -> B_dist2 -> B_dist1 -> B_dist1)
               pattern, written out for 16 frames in groups of 8 and 4, and a processing order
               that puts every frame after its references
  reorder_future     a B frame equal to its future anchor reuses from it at every layer and
               copies its outputs; swapping the anchors' roles swaps the source
  reorder_brute      == the per-token loop implementation (gate and injection modes, with
               restoration and with the decision MLP, groups of 4, 8 and 12, short last groups)
"""
import numpy as np

import synth
from synth.configs import ModelConfig

from oracle.bruteforce import encode_bruteforce
from oracle.dense_vit import dense_vit

from . import torch_ref

M_A = ModelConfig(32, 16, 2, 8, 2, 16, "f32")       # N=5, D=8, L=2
M_B = ModelConfig(48, 16, 2, 16, 2, 32, "f32")      # N=10, D=16, L=2
M_1 = ModelConfig(48, 16, 1, 16, 2, 32, "f32")      # one layer
M_AR = ModelConfig(32, 16, 2, 8, 2, 16, "f32", restore=True)     # M_A with restoration
M_BR = ModelConfig(48, 16, 2, 16, 2, 32, "f32", restore=True)    # M_B with restoration
M_1R = ModelConfig(48, 16, 1, 16, 2, 32, "f32", restore=True)    # M_1 with restoration
M_AD = ModelConfig(32, 16, 2, 8, 2, 16, "f32", decision=True)    # M_A with the decision MLP
M_BD = ModelConfig(48, 16, 2, 16, 2, 32, "f32", decision=True)   # M_B with the decision MLP
M_BRD = ModelConfig(48, 16, 2, 16, 2, 32, "f32", restore=True, decision=True)


def weights(m, seed=7, perturb=True):
    w = synth.make_weights(m, seed, perturb_ln=perturb, std=0.3)
    return w, synth.pack_weights(w, m)


def mixed_frames(m, F, G, seed=11):
    """Groups whose non-reference frames copy the reference patch-wise, with a random half of
    the patches perturbed by noise of mixed strength (so cosines spread over [-1, 1])."""
    rng = np.random.default_rng(seed)
    S, p = m.image_size, m.patch
    g = S // p
    fr = np.empty((F, 3, S, S), np.float32)
    for f in range(F):
        if f % G == 0:
            fr[f] = rng.standard_normal((3, S, S))
            base = fr[f].copy()
            continue
        fr[f] = base
        for r in range(g):
            for c in range(g):
                if rng.random() < 0.5:
                    amp = rng.choice([0.05, 0.3, 1.0, 3.0])
                    fr[f, :, r * p:(r + 1) * p, c * p:(c + 1) * p] += \
                        amp * rng.standard_normal((3, p, p))
    return fr


def _close(a, b, tol, what):
    a, b = np.asarray(a), np.asarray(b)
    assert a.shape == b.shape, f"{what}: shape {a.shape} vs {b.shape}"
    err = np.max(np.abs(a - b)) if a.size else 0.0
    assert err <= tol, f"{what}: max abs diff {err:.3e} > {tol:.1e}"


def assert_copy(r, f, ref):
    """Frame f copies frame ref: reused rows bitwise; the class token, recomputed from an equal
    input against equal keys/values, to rounding (BLAS may order a 1-row product differently
    from a full-frame one)."""
    assert np.array_equal(r["tokens"][f, 1:], r["tokens"][ref, 1:]), f"frame {f} rows not a copy"
    _close(r["tokens"][f, 0], r["tokens"][ref, 0], 1e-12, f"frame {f} class token")
    _close(r["emb"][f], r["emb"][ref], 1e-12, f"frame {f} embedding")


def pin_library(ora):
    for m in (M_A, M_B):
        w, blob = weights(m)
        fr = mixed_frames(m, 4, 4)
        e_t, x_t = torch_ref.vit(fr, w, m)
        r = ora.encode(fr, blob, m.as_dict(), 4, tau=-np.inf)
        _close(r["tokens"], x_t, 1e-10, "tokens vs torch")
        _close(r["emb"], e_t, 1e-10, "embeddings vs torch")


def pin_dense_vit(ora):
    m = M_B
    w, blob = weights(m, 3)
    fr = mixed_frames(m, 6, 3)
    e, x = dense_vit(fr, blob, m.as_dict(), return_tokens=True)
    r = ora.encode(fr, blob, m.as_dict(), 3, tau=-np.inf)
    _close(r["emb"], e, 1e-11, "emb vs dense_vit")
    _close(r["tokens"], x, 1e-11, "tokens vs dense_vit")
    assert not r["masks"].any()


def pin_bruteforce(ora):
    for m, G in ((M_A, 4), (M_B, 3)):
        w, blob = weights(m, 5)
        fr = mixed_frames(m, 7, G, seed=5)
        cfg = m.as_dict()
        for tau in (-np.inf, 0.3, 0.8, 0.97, np.inf):
            r = ora.encode(fr, blob, cfg, G, tau=tau)
            b = encode_bruteforce(fr, blob, cfg, G, tau=tau)
            assert np.array_equal(r["masks"], b["masks"]), f"masks differ at tau={tau}"
            _close(r["tokens"], b["tokens"], 1e-12, f"tokens tau={tau}")
            _close(r["emb"], b["emb"], 1e-12, f"emb tau={tau}")
        rng = np.random.default_rng(9)
        mk = (rng.random((7, m.depth, m.n_tokens)) < 0.5).astype(np.uint8)
        r = ora.encode(fr, blob, cfg, G, masks=mk)
        b = encode_bruteforce(fr, blob, cfg, G, masks=mk)
        assert np.array_equal(r["masks"], b["masks"]), "effective injected masks differ"
        _close(r["tokens"], b["tokens"], 1e-12, "tokens (injected)")


def pin_copy(ora):
    m = M_B
    _, blob = weights(m, 8)
    G = 4
    fr = mixed_frames(m, 8, G, seed=8)
    r = ora.encode(fr, blob, m.as_dict(), G, tau=np.inf)
    for f in range(8):
        ref = (f // G) * G
        assert_copy(r, f, ref)
        if f != ref:
            assert r["masks"][f, :, 1:].all() and not r["masks"][f, :, 0].any()


def pin_ref_dense(ora):
    m = M_B
    _, blob = weights(m, 12)
    G = 3
    fr = mixed_frames(m, 7, G, seed=12)
    e = dense_vit(fr, blob, m.as_dict())
    for tau in (0.2, 0.9, np.inf):
        r = ora.encode(fr, blob, m.as_dict(), G, tau=tau)
        for f in range(0, 7, G):
            _close(r["emb"][f], e[f], 1e-11, f"reference frame {f}")
            assert not r["masks"][f].any()
        assert not r["masks"][:, :, 0].any(), "class token must never be reused"


def pin_monotone(ora):
    m = M_B
    _, blob = weights(m, 13)
    fr = mixed_frames(m, 8, 4, seed=13)
    seen_reuse = False
    for tau in (0.3, 0.7, 0.95, 0.999, 1.0):
        mk = ora.encode(fr, blob, m.as_dict(), 4, tau=tau)["masks"]
        assert np.all(mk[:, 1:] >= mk[:, :-1]), f"reuse not monotone over layers at tau={tau}"
        seen_reuse |= bool(mk.any())
    assert seen_reuse


def pin_static(ora):
    m = M_B
    _, blob = weights(m, 14)
    one = mixed_frames(m, 1, 1, seed=14)
    fr = np.repeat(one, 4, axis=0)
    for tau in (-0.5, 0.5, 0.99, 1.0):
        r = ora.encode(fr, blob, m.as_dict(), 4, tau=tau)
        assert r["masks"][1:, :, 1:].all(), f"static video not fully reused at tau={tau}"
        for f in range(1, 4):
            assert_copy(r, f, 0)
    r = ora.encode(fr, blob, m.as_dict(), 4, tau=1.0 + 1e-9)
    assert not r["masks"].any(), "tau above 1 must reuse nothing"


def pin_g1(ora):
    m = M_B
    _, blob = weights(m, 15)
    fr = mixed_frames(m, 5, 2, seed=15)
    e = dense_vit(fr, blob, m.as_dict())
    r = ora.encode(fr, blob, m.as_dict(), 1, tau=-1.0)
    _close(r["emb"], e, 1e-11, "G=1")
    assert not r["masks"].any()


def pin_groups(ora):
    m = M_B
    _, blob = weights(m, 16)
    G = 3
    fr = mixed_frames(m, 9, G, seed=16)
    cfg = m.as_dict()
    a = ora.encode(fr, blob, cfg, G, tau=0.8)
    perm = [2, 0, 1]
    fr_p = np.concatenate([fr[g * G:(g + 1) * G] for g in perm])
    b = ora.encode(fr_p, blob, cfg, G, tau=0.8)
    for k, g in enumerate(perm):
        assert np.array_equal(b["emb"][k * G:(k + 1) * G], a["emb"][g * G:(g + 1) * G])
        assert np.array_equal(b["masks"][k * G:(k + 1) * G], a["masks"][g * G:(g + 1) * G])
    c1 = ora.encode(fr[:6], blob, cfg, G, tau=0.8)
    c2 = ora.encode(fr[6:], blob, cfg, G, tau=0.8)
    assert np.array_equal(np.concatenate([c1["emb"], c2["emb"]]), a["emb"])


def pin_inject_one(ora):
    m = M_1
    w, blob = weights(m, 17)
    fr = mixed_frames(m, 2, 2, seed=17)
    j = 4
    mk = np.zeros((2, 1, m.n_tokens), np.uint8)
    mk[1, 0, j] = 1
    r = ora.encode(fr, blob, m.as_dict(), 2, masks=mk, return_layers=True)
    x0 = torch_ref.embed(fr, w, m).numpy()
    _close(r["layers"][0], x0, 1e-12, "layer input vs conv2d embedding")
    ref_out = torch_ref.layer_with_substituted_kv(x0[0], x0[0], j, w, 0, m)
    f_out = torch_ref.layer_with_substituted_kv(x0[1], x0[0], j, w, 0, m)
    y = r["layers"][1]
    _close(y[0], ref_out, 1e-11, "reference frame layer output")
    assert np.array_equal(y[1, j], y[0, j]), "reused row must copy the reference output"
    rows = [i for i in range(m.n_tokens) if i != j]
    _close(y[1, rows], f_out[rows], 1e-11, "other queries with the reference's K/V at j")


def pin_extremes(ora):
    m = M_B
    _, blob = weights(m, 18)
    fr = mixed_frames(m, 8, 4, seed=18)
    cfg = m.as_dict()
    lo, hi = ora.encode(fr, blob, cfg, 4, tau=-np.inf), ora.encode(fr, blob, cfg, 4, tau=2.0)
    assert np.array_equal(lo["tokens"], hi["tokens"]) and not hi["masks"].any()
    a, b = ora.encode(fr, blob, cfg, 4, tau=np.inf), ora.encode(fr, blob, cfg, 4, tau=-2.0)
    assert np.array_equal(a["tokens"], b["tokens"])
    assert np.array_equal(a["masks"], b["masks"])


def pin_star(ora):
    m = M_B
    _, blob = weights(m, 19)
    fr = mixed_frames(m, 4, 4, seed=19)
    fr[2] = fr[0]                 # frame 2 repeats the group's first frame exactly
    r = ora.encode(fr, blob, m.as_dict(), 4, tau=0.9999)
    assert r["masks"][2, :, 1:].all(), "frame equal to the reference must be fully reused"
    assert_copy(r, 2, 0)
    assert not r["masks"][1, 0, 1:].all(), "frame 1 differs from the reference"


def pin_cosine(ora):
    th = np.linspace(0.0, np.pi, 7)
    a = np.stack([np.ones_like(th), np.zeros_like(th), np.zeros_like(th)], 1) * 2.5
    b = np.stack([np.cos(th), np.sin(th), np.zeros_like(th)], 1) * 0.7
    c = ora.cosine_rows(a, b)
    assert np.allclose(c, np.cos(th), atol=1e-15, rtol=0), f"cosine {c} vs {np.cos(th)}"
    assert ora.cosine_rows(a, -a)[0] == -1.0
    v = np.random.default_rng(1).standard_normal((5, 9))
    assert np.all(ora.cosine_rows(v, v) == 1.0), "equal rows must give exactly 1"
    z = np.zeros((1, 4))
    assert ora.cosine_rows(z, z)[0] == 1.0
    assert ora.cosine_rows(z, np.ones((1, 4)))[0] == 0.0
    cs = np.array([0.5, 0.94999, 0.95, 0.96])
    assert list(ora.gate_decision(cs, 0.95)) == [False, False, True, True], "tie must reuse"


def pin_partial(ora):
    m = M_B
    _, blob = weights(m, 20)
    fr = mixed_frames(m, 6, 4, seed=20)
    e = dense_vit(fr, blob, m.as_dict())
    r = ora.encode(fr, blob, m.as_dict(), 4, tau=np.inf)
    _close(r["emb"][4], e[4], 1e-11, "first frame of the short last group")
    assert_copy(r, 5, 4)


def pin_rate(ora):
    mk = np.zeros((6, 2, 5), np.uint8)
    mk[1, 0, 1:3] = 1       # 2 reused
    mk[5, 1, :] = 1         # 5 reused (a reference frame's entries would not count)
    mk[4, 1, :] = 1         # frame 4 is a reference at G=4: not counted
    # non-reference frames at G=4: 1, 2, 3, 5 -> denominator 4 * 2 * 5 = 40
    assert abs(ora.reuse_rate(mk, 4) - 7 / 40) < 1e-15


def _without_restoration(w, m):
    """The blob of the same weights and the model without the restoration section."""
    base = ModelConfig(m.image_size, m.patch, m.depth, m.width, m.heads, m.mlp, m.dtype)
    return base, synth.pack_weights(w, base)


def pin_restore_zero(ora):
    m = M_BR
    w, _ = weights(m, 21)
    for l in range(m.depth):
        w[f"l{l}.W_r2"][...] = 0.0
        w[f"l{l}.b_r2"][...] = 0.0
    blob = synth.pack_weights(w, m)
    base, blob0 = _without_restoration(w, m)
    fr = mixed_frames(m, 8, 4, seed=21)
    for tau in (0.5, 0.9, np.inf):
        a = ora.encode(fr, blob, m.as_dict(), 4, tau=tau)
        b = ora.encode(fr, blob0, base.as_dict(), 4, tau=tau)
        assert np.array_equal(a["masks"], b["masks"]), f"masks differ at tau={tau}"
        assert np.array_equal(a["tokens"], b["tokens"]), f"tokens differ at tau={tau}"


def pin_restore_brute(ora):
    for m, G in ((M_AR, 4), (M_BR, 3)):
        _, blob = weights(m, 24)
        fr = mixed_frames(m, 7, G, seed=24)
        cfg = m.as_dict()
        for tau in (0.3, 0.8, 0.97, np.inf):
            r = ora.encode(fr, blob, cfg, G, tau=tau)
            b = encode_bruteforce(fr, blob, cfg, G, tau=tau)
            assert np.array_equal(r["masks"], b["masks"]), f"masks differ at tau={tau}"
            _close(r["tokens"], b["tokens"], 1e-12, f"tokens tau={tau}")
        mk = (np.random.default_rng(25).random((7, m.depth, m.n_tokens)) < 0.5).astype(np.uint8)
        r = ora.encode(fr, blob, cfg, G, masks=mk)
        b = encode_bruteforce(fr, blob, cfg, G, masks=mk)
        _close(r["tokens"], b["tokens"], 1e-12, "tokens (injected)")


def pin_restore_one(ora):
    m = M_1R
    w, blob = weights(m, 22)
    base, blob0 = _without_restoration(w, m)
    fr = mixed_frames(m, 2, 2, seed=22)
    j = 4
    mk = np.zeros((2, 1, m.n_tokens), np.uint8)
    mk[1, 0, j] = 1
    r = ora.encode(fr, blob, m.as_dict(), 2, masks=mk, return_layers=True)
    r0 = ora.encode(fr, blob0, base.as_dict(), 2, masks=mk, return_layers=True)
    x0 = torch_ref.embed(fr, w, m).numpy()
    dx = (x0[1, j] - x0[0, j])[None]
    want = r0["layers"][1][0, j] + torch_ref.restoration(dx, w, 0)[0]
    _close(r["layers"][1][1, j], want, 1e-12, "restored row")
    y, y0 = r["layers"][1].copy(), r0["layers"][1].copy()
    y[1, j] = y0[1, j] = 0.0
    assert np.array_equal(y, y0), "restoration must touch only the reused row"


def pin_restore_static(ora):
    m = M_BR
    w, blob = weights(m, 23)
    fr = np.repeat(mixed_frames(m, 1, 1, seed=23), 3, axis=0)
    r = ora.encode(fr, blob, m.as_dict(), 3, tau=np.inf, return_layers=True)
    D = m.width
    c0 = torch_ref.restoration(np.zeros((1, D)), w, 0)[0]      # layer 0: equal inputs
    x1, x2 = r["layers"][1], r["layers"][2]
    for f in (1, 2):
        _close(x1[f, 1:] - x1[0, 1:], np.broadcast_to(c0, x1[0, 1:].shape), 1e-12,
               f"layer 0 restored rows, frame {f}")
        _close(x1[f, 0], x1[0, 0], 1e-12, f"layer 0 class token, frame {f}")
        d = x1[f, 1:] - x1[0, 1:]                               # layer 1: input difference c0
        _close(x2[f, 1:] - x2[0, 1:], torch_ref.restoration(d, w, 1), 1e-12,
               f"layer 1 restored rows, frame {f}")


def linear_decision(w, m, col, a, theta, c=40.0):
    """Make every layer's decision MLP the affine function d = a * (v[col] - theta) of one
    input feature: hidden unit 0 computes a * v[col] + c, where GELU is the identity to fp64
    rounding (erf(c / sqrt 2) rounds to 1 for c > 8.4), the other units are switched off.
    Returns the blob and the threshold the fp32 weights hold (theta after rounding)."""
    for l in range(m.depth):
        for k in ("W_d1", "b_d1", "W_d2", "b_d2"):
            w[f"l{l}.{k}"][...] = 0.0
        w[f"l{l}.W_d1"][0, col] = a
        w[f"l{l}.b_d1"][0] = c
        w[f"l{l}.W_d2"][0, 0] = 1.0
        w[f"l{l}.b_d2"][0] = -c - a * theta
    held = (-float(w["l0.b_d2"][0]) - c) / a
    return synth.pack_weights(w, m), held


def _without_decision(w, m):
    base = ModelConfig(m.image_size, m.patch, m.depth, m.width, m.heads, m.mlp, m.dtype,
                       restore=m.restore)
    return base, synth.pack_weights(w, base)


def pin_decision_threshold(ora):
    m = M_BD
    w, _ = weights(m, 31)
    base, blob0 = _without_decision(w, m)
    fr = mixed_frames(m, 8, 4, seed=31)
    for theta in (0.3, 0.8, 0.95):
        want = ora.encode(fr, blob0, base.as_dict(), 4, tau=theta)
        c = want["cos"][~np.isnan(want["cos"])]
        assert np.min(np.abs(c - theta)) > 1e-9, "threshold too close to a cosine"
        blob, th = linear_decision(w, m, 0, 5.0, theta)
        assert np.min(np.abs(c - th)) > 1e-9
        r = ora.encode(fr, blob, m.as_dict(), 4, tau=0.0)
        assert np.array_equal(r["masks"], want["masks"]), f"maps differ at theta={theta}"
        assert np.array_equal(r["tokens"], want["tokens"]), f"tokens differ at theta={theta}"
        ev = ~np.isnan(r["cos"])
        _close(r["dec"][ev], 5.0 * (r["cos"][ev] - th), 1e-12, "decision values")


def pin_decision_attention(ora):
    m = M_BD
    N = m.n_tokens
    w, _ = weights(m, 32)
    fr = mixed_frames(m, 4, 4, seed=32)
    x0 = torch_ref.embed(fr, w, m).numpy()
    t0 = [torch_ref.cls_attention(x0[f], x0[f], w, 0, m) for f in range(4)]
    # threshold above the first layer's uniform 1/N: nothing reused at layer 0
    blob, theta = linear_decision(w, m, 1, 1.0, 1.02 / N)
    assert min(np.min(np.abs(t[1:] - theta)) for t in t0[1:]) > 1e-9
    r = ora.encode(fr, blob, m.as_dict(), 4, tau=0.0)
    assert not r["masks"][:, 0].any(), "t = 1/N at the first layer"
    _close(r["dec"][1:, 0, 1:], np.full((3, N - 1), 1.0 / N - theta), 1e-12, "layer-0 decisions")
    for f in (1, 2, 3):   # layer 1: the class token's attention in frame f's (dense) layer 0
        _close(r["dec"][f, 1, 1:], t0[f][1:] - theta, 1e-12, f"layer-1 decisions, frame {f}")
        assert np.array_equal(r["masks"][f, 1, 1:] != 0, t0[f][1:] > theta)
    assert 0 < r["masks"][:, 1].mean() < 0.75, "want a mixed map at layer 1"
    # an injected reuse at layer 0: the class query of frame 1 sees the reference's key/value
    j = 3
    mk = np.zeros((4, m.depth, N), np.uint8)
    mk[1, 0, j] = 1
    r = ora.encode(fr, blob, m.as_dict(), 4, masks=mk)
    xs = x0[1].copy()
    xs[j] = x0[0, j]
    t = torch_ref.cls_attention(x0[1], xs, w, 0, m)
    _close(r["dec"][1, 1, 1:], t[1:] - theta, 1e-12, "layer-1 decisions after an injected reuse")
    # below 1/N: everything reused at layer 0
    blob, _ = linear_decision(w, m, 1, 1.0, 0.98 / N)
    r = ora.encode(fr, blob, m.as_dict(), 4, tau=0.0)
    assert r["masks"][1:, 0, 1:].all() and not r["masks"][:, :, 0].any()


def pin_decision_type(ora):
    m = M_BD
    w, _ = weights(m, 33)
    fr = mixed_frames(m, 6, 3, seed=33)
    cfg = m.as_dict()
    cases = ((3, 0.5, np.inf),      # P entry: d = +0.5 for every non-reference token
             (2, 0.5, -np.inf),     # I entry: d = -0.5
             (3, 1.0, -np.inf))     # P entry, d == 0 exactly: the tie recomputes
    for col, theta, same_as in cases:
        blob, _ = linear_decision(w, m, col, 1.0, theta)
        r = ora.encode(fr, blob, cfg, 3, tau=0.0)
        want = ora.encode(fr, blob, cfg, 3, tau=same_as)
        assert np.array_equal(r["masks"], want["masks"]), f"maps (column {col}, theta {theta})"
        assert np.array_equal(r["tokens"], want["tokens"]), f"tokens (column {col})"
    ev = ~np.isnan(r["dec"])
    assert ev.any() and np.all(r["dec"][ev] == 0.0)


def pin_decision_mlp(ora):
    m = M_BD
    N = m.n_tokens
    w, blob = weights(m, 34)
    fr = mixed_frames(m, 6, 3, seed=34)
    r = ora.encode(fr, blob, m.as_dict(), 3, tau=0.0)
    x0 = torch_ref.embed(fr, w, m).numpy()
    for f in (1, 2, 4, 5):
        a, b = x0[f, 1:], x0[f - f % 3, 1:]
        s = np.sum(a * b, 1) / (np.linalg.norm(a, axis=1) * np.linalg.norm(b, axis=1))
        v = np.zeros((N - 1, 6))
        v[:, 0], v[:, 1], v[:, 3] = s, 1.0 / N, 1.0
        _close(r["dec"][f, 0, 1:], torch_ref.decision_mlp(v, w, 0), 1e-12, f"frame {f}")
    dv = r["dec"][~np.isnan(r["dec"])]
    assert np.ptp(dv) > 0.1, "decision values should spread"


def pin_decision_brute(ora):
    for m, G in ((M_AD, 4), (M_BD, 3), (M_BRD, 3)):
        w, blob = weights(m, 35)
        fr = mixed_frames(m, 7, G, seed=35)
        cfg = m.as_dict()
        r0 = ora.encode(fr, blob, cfg, G, tau=0.0)
        dv = r0["dec"][~np.isnan(r0["dec"])]
        for tau in (np.quantile(dv, 0.3), np.quantile(dv, 0.7), np.inf, -np.inf):
            tau = float(tau)
            r = ora.encode(fr, blob, cfg, G, tau=tau)
            b = encode_bruteforce(fr, blob, cfg, G, tau=tau)
            assert np.array_equal(r["masks"], b["masks"]), f"masks differ at tau={tau}"
            _close(r["tokens"], b["tokens"], 1e-12, f"tokens tau={tau}")
            _close(r["emb"], b["emb"], 1e-12, f"emb tau={tau}")


M_BO = ModelConfig(48, 16, 2, 16, 2, 32, "f32")   # M_B, run with cfg["reorder"]


def reorder_cfg(m):
    import dataclasses
    return dataclasses.replace(m, reorder=True).as_dict()


# the paper's pattern, frames 0..15: (type, past reference, future reference), types
# 0 I, 1 P, 2 B_dist2, 3 B_dist1
PATTERN_G8 = [(0, None, None), (3, 0, 2), (2, 0, 4), (3, 2, 4), (1, 0, None), (3, 4, 6),
              (2, 4, 8), (3, 6, 8), (0, None, None), (3, 8, 10), (2, 8, 12), (3, 10, 12),
              (1, 8, None), (3, 12, 14), (2, 12, None), (3, 14, None)]
PATTERN_G4 = [(0, None, None), (3, 0, 2), (2, 0, 4), (3, 2, 4), (0, None, None), (3, 4, 6),
              (2, 4, 8), (3, 6, 8), (0, None, None), (3, 8, 10), (2, 8, 12), (3, 10, 12),
              (0, None, None), (3, 12, 14), (2, 12, None), (3, 14, None)]


def pin_reorder_pattern(ora):
    for G, want in ((8, PATTERN_G8), (4, PATTERN_G4)):
        got = [ora.reference_frames(f, G, 16) for f in range(16)]
        assert got == want, f"reference graph, groups of {G}: {got}"
        order = ora.processing_order(16, G)
        assert sorted(order) == list(range(16))
        at = {f: k for k, f in enumerate(order)}
        for f, (_, a, b) in enumerate(got):
            assert all(at[r] < at[f] for r in (a, b) if r is not None), f"frame {f} before a ref"
    assert ora.processing_order(16, 8)[:5] == [0, 4, 2, 1, 3]
    # groups of 12: a chain of P frames, each referencing the anchor four frames back
    assert [ora.reference_frames(f, 12, 14)[:2] for f in (4, 8, 12)] == [(1, 0), (1, 4), (0, None)]
    assert ora.reference_frames(10, 12, 14) == (2, 8, 12)


def pin_reorder_future(ora):
    m = M_BO
    w, blob = weights(m, 36)
    fr = mixed_frames(m, 9, 8, seed=36)
    fr[4] = np.random.default_rng(37).standard_normal(fr[4].shape)   # the P anchor: a new scene
    fr[2] = fr[4]                                                      # B_dist2 == future anchor
    for tau in (0.9, np.inf):
        r = ora.encode(fr, blob, reorder_cfg(m), 8, tau=tau)
        assert r["masks"][2, :, 1:].all(), "every token of frame 2 reused"
        # at layer 0 from the future anchor (later, where the anchor itself copied frame 0,
        # both references hold equal rows and the tie takes the past one)
        assert (r["src"][2, 0, 1:] == 1).all(), "... from its future anchor"
        assert_copy(r, 2, 4)
    # the mirror case: frame 2 equal to its past anchor (frame 0) reuses from the past
    fr = mixed_frames(m, 9, 8, seed=38)
    fr[4] = np.random.default_rng(39).standard_normal(fr[4].shape)
    fr[2] = fr[0]
    r = ora.encode(fr, blob, reorder_cfg(m), 8, tau=0.9)
    assert r["masks"][2, :, 1:].all() and (r["src"][2, :, 1:] == 0).all()
    assert_copy(r, 2, 0)


def pin_reorder_brute(ora):
    cases = ((M_A, 4, 11), (M_B, 8, 13), (M_B, 12, 14), (M_BR, 4, 9), (M_BD, 8, 10),
             (M_BRD, 4, 9))
    for m, G, F in cases:
        w, blob = weights(m, 40 + G)
        fr = mixed_frames(m, F, G, seed=F)
        cfg = reorder_cfg(m)
        taus = (0.0, 1.0, 2.0) if m.decision else (0.3, 0.8, 0.97, np.inf)
        for tau in taus:
            r = ora.encode(fr, blob, cfg, G, tau=tau)
            b = encode_bruteforce(fr, blob, cfg, G, tau=tau)
            assert np.array_equal(r["masks"], b["masks"]), f"masks differ at tau={tau}"
            _close(r["tokens"], b["tokens"], 1e-12, f"tokens tau={tau}")
            _close(r["emb"], b["emb"], 1e-12, f"emb tau={tau}")
        mk = (np.random.default_rng(F).random((F, m.depth, m.n_tokens)) < 0.6).astype(np.uint8)
        r = ora.encode(fr, blob, cfg, G, masks=mk)
        b = encode_bruteforce(fr, blob, cfg, G, masks=mk)
        assert np.array_equal(r["masks"], b["masks"]), "effective injected masks differ"
        _close(r["tokens"], b["tokens"], 1e-12, "tokens (injected)")


ALL_PINS = [pin_library, pin_dense_vit, pin_bruteforce, pin_copy, pin_ref_dense, pin_monotone,
            pin_static, pin_g1, pin_groups, pin_inject_one, pin_extremes, pin_star, pin_cosine,
            pin_partial, pin_rate, pin_restore_zero, pin_restore_brute, pin_restore_one,
            pin_restore_static, pin_decision_threshold, pin_decision_attention, pin_decision_type,
            pin_decision_mlp, pin_decision_brute, pin_reorder_pattern, pin_reorder_future,
            pin_reorder_brute]
