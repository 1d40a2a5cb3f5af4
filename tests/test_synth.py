"""Seeded input generators: determinism, blob layout agreement, recipe structure."""
import numpy as np

import synth
from oracle.reusevit import unpack_blob
from synth.configs import ModelConfig, Segment, VideoRecipe


def test_blob_layout_matches_oracle_reader():
    m = ModelConfig(48, 16, 3, 16, 2, 40, "f32")
    w = synth.make_weights(m, 1, perturb_ln=True)
    blob = synth.pack_weights(w, m)
    assert blob.size == synth.weights.blob_floats(m)
    W = unpack_blob(blob, m.as_dict())
    assert np.array_equal(W["W_pe"], w["W_pe"]) and np.array_equal(W["pos"], w["pos"])
    for l in range(m.depth):
        for k in ("ln1_g", "ln1_b", "W_qkv", "b_qkv", "W_o", "b_o", "ln2_g", "ln2_b",
                  "W_1", "b_1", "W_2", "b_2"):
            assert np.array_equal(W["layers"][l][k], w[f"l{l}.{k}"]), (l, k)
    assert np.array_equal(W["lnf_g"], w["lnf_g"])
    assert np.array_equal(synth.make_blob(m, 1, perturb_ln=True), blob)


def test_weights_deterministic_and_bf16():
    m = ModelConfig(32, 16, 1, 16, 2, 32, "bf16")
    a = synth.make_blob(m, 3)
    b = synth.make_blob(m, 3)
    assert np.array_equal(a, b)
    assert not np.array_equal(a, synth.make_blob(m, 4))
    assert np.all((a.view(np.uint32) & 0xFFFF) == 0), "bf16 weights must be bf16-representable"
    w = synth.make_weights(m, 3)
    assert np.all(w["l0.ln1_g"] == 1) and np.all(w["l0.ln1_b"] == 0)
    assert 0.015 < np.std(w["l0.W_qkv"]) < 0.025


def test_round_to_bf16_ties_even():
    x = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -9, -3.0], np.float32)
    y = synth.round_to_bf16(x)
    assert list(y) == [1.0, 1.0, 1 + 2 ** -6, 1.0, -3.0]


def test_frames_lazy_equals_batch_and_deterministic():
    rec = synth.get_config("vit_l14").video
    a = synth.render_frames(rec, 56, 0, 6)
    b = np.stack([synth.render_frame(rec, 56, t) for t in range(6)])
    assert np.array_equal(a, b)
    assert np.array_equal(synth.render_frames(rec, 56, 3, 2), a[3:5])
    assert a.dtype == np.float32 and a.shape == (6, 3, 56, 56)


def test_static_recipe_gives_identical_frames():
    rec = VideoRecipe(seed=5, sigma=0.0, segments=(Segment(1 << 30, 3, 8, 0.0, 0.0),))
    fr = synth.render_frames(rec, 32, 0, 4)
    assert all(np.array_equal(fr[0], fr[k]) for k in range(4))


def test_scene_cuts_fall_mid_group():
    w = synth.get_config("vit_l14_336")
    rec = w.video
    S = 112
    f = synth.render_frames(rec, S, 58, 4)            # frames 58..61, cut at 60
    d_same = np.abs(f[1] - f[0]).mean()
    d_cut = np.abs(f[2] - f[1]).mean()
    assert d_cut > 2 * d_same
    assert rec.cut_first % w.group_size != 0


def test_pan_moves_background():
    rec = VideoRecipe(seed=5, sigma=0.0, segments=(Segment(1 << 30, 0, 8, 0.0, 1.0),))
    fr = synth.render_frames(rec, 32, 0, 2)
    # the background shifts left by one pixel per frame (periodic wrap)
    assert np.allclose(fr[1][:, :, :-1], fr[0][:, :, 1:], atol=1e-5)
