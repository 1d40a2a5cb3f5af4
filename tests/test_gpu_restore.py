"""The restoration layer on reused rows (Section 3.3) through the C ABI against the CPU oracle:
gate mode (teacher-forced decisions), mask injection, and a zero output layer reproducing the
path without restoration bitwise."""
import dataclasses

import numpy as np
import pytest

import oracle
import synth
from synth.configs import ModelConfig

from .gpu_util import check_close, dev, encoder, host, mask_parity, require_gpu
from .test_gpu_parity import _video

pytestmark = pytest.mark.gpu

TINY = synth.get_config("tiny")
TINY_R = dataclasses.replace(TINY.model, restore=True)
SMALL_R = ModelConfig(64, 16, 2, 128, 2, 256, "bf16", restore=True)
MID_R = ModelConfig(112, 16, 3, 256, 4, 512, "bf16", restore=True)


def _weights(m, seed, std=0.02):
    return synth.make_weights(m, seed, perturb_ln=True, std=std)


def test_tiny_restore_gate_mode():
    torch = require_gpu()
    m = TINY_R
    w = _weights(m, TINY.weight_seed, std=0.05)
    blob = synth.pack_weights(w, m)
    fr = synth.render_frames(TINY.video, m.image_size, 0, TINY.n_frames)
    tau = float(np.float32(TINY.tau))
    emb, masks, toks = encoder(m, blob, 8).encode(dev(fr), 4, tau, want_tokens=True)
    torch.cuda.synchronize()
    mg = host(masks)
    r = oracle.encode(fr, blob, m.as_dict(), 4, masks=mg)   # teacher-forced decisions
    bad, _ = mask_parity(mg, r["cos"], tau)
    assert bad == 0, f"{bad} decisions differ outside the 1e-3 band"
    check_close(host(emb), r["emb"], "f32", "embeddings")
    check_close(host(toks), r["tokens"], "f32", "tokens")
    assert 0.1 < oracle.reuse_rate(mg, 4) < 1.0
    # the restoration changes the reused rows: the run without it differs
    base = dataclasses.replace(m, restore=False)
    r0 = oracle.encode(fr, synth.pack_weights(w, base), base.as_dict(), 4, masks=mg)
    assert np.max(np.abs(r0["tokens"] - r["tokens"])) > 1e-3


@pytest.mark.parametrize("m", [SMALL_R, MID_R], ids=["small", "mid"])
def test_bf16_restore_injection(m):
    torch = require_gpu()
    w = _weights(m, 31, std=0.05)
    blob = synth.pack_weights(w, m)
    F, G = 9, 4                                  # a short last group
    fr = _video(m, F, seed=31)
    mk = (np.random.default_rng(32).random((F, m.depth, m.n_tokens)) < 0.6).astype(np.uint8)
    emb, eff, toks = encoder(m, blob, 8).encode_masked(dev(fr), G, dev(mk), want_tokens=True)
    torch.cuda.synchronize()
    r = oracle.encode(fr, blob, m.as_dict(), G, masks=mk)
    assert np.array_equal(host(eff), r["masks"]), "effective maps"
    check_close(host(emb), r["emb"], "bf16", "embeddings")
    check_close(host(toks), r["tokens"], "bf16", "tokens")


@pytest.mark.parametrize("m,tau", [(TINY_R, 0.95), (SMALL_R, 0.9)], ids=["tiny", "small"])
def test_restore_zero_output_layer_is_no_restoration(m, tau):
    torch = require_gpu()
    w = _weights(m, 33)
    for l in range(m.depth):
        w[f"l{l}.W_r2"][...] = 0.0
        w[f"l{l}.b_r2"][...] = 0.0
    base = dataclasses.replace(m, restore=False)
    F, G = 8, 4
    fr = _video(m, F, seed=33)
    tau = float(np.float32(tau))
    out = []
    for mm in (m, base):
        e, k, t = encoder(mm, synth.pack_weights(w, mm), 8).encode(dev(fr), G, tau,
                                                                   want_tokens=True)
        torch.cuda.synchronize()
        out.append((host(e), host(k), host(t)))
    assert out[0][1].any(), "some tokens must be reused"
    for a, b, what in zip(out[0], out[1], ("embeddings", "masks", "tokens")):
        assert np.array_equal(a, b), f"{what} differ"
