"""HIP path (through the C ABI) against the CPU oracle: masks, embeddings, token buffers,
stream compaction, exact-copy and determinism properties, edge cases."""
import numpy as np
import pytest

import oracle
import synth
from synth.configs import ModelConfig

from .gpu_util import (check_close, dev, encoder, host, mask_parity, require_gpu)

pytestmark = pytest.mark.gpu

TINY = synth.get_config("tiny")
# a small bf16 model: N = 17 tokens, D = 128, two heads of 64, two layers
SMALL_BF16 = ModelConfig(64, 16, 2, 128, 2, 256, "bf16")
# N = 50 tokens in bf16 with three layers
MID_BF16 = ModelConfig(112, 16, 3, 256, 4, 512, "bf16")
# ViT-L/14 token counts (257 at 224 px, 577 at 336 px) with a narrow width
N257_BF16 = ModelConfig(224, 14, 2, 128, 2, 256, "bf16")
N577_BF16 = ModelConfig(336, 14, 1, 128, 2, 256, "bf16")
# head dim 80 (the ViT-H/14-class width 1280 / 16 heads)
DH80_BF16 = ModelConfig(64, 16, 2, 640, 8, 1280, "bf16")
# head dim 80 with two key blocks per frame (N = 50): the per-frame attention kernel
DH80_N50 = ModelConfig(112, 16, 2, 640, 8, 1280, "bf16")
# widths past 1024 that the row kernels hold as five float4 chunks per lane: 1152 (the last
# chunk on half of the lanes) and 1280 (the ViT-H/14-class width)
W1152_BF16 = ModelConfig(64, 16, 2, 1152, 18, 2304, "bf16")
W1280_BF16 = ModelConfig(64, 16, 2, 1280, 16, 2560, "bf16")


def _video(m, n, seed=2000, sigma=0.01, speed=3.0, n_obj=2, size=None, pan=0.0):
    rec = synth.VideoRecipe(seed=seed, sigma=sigma, segments=(
        synth.configs.Segment(1 << 30, n_obj, size or max(4, m.image_size // 7), speed, pan),))
    return synth.render_frames(rec, m.image_size, 0, n)


def _tiny():
    m = TINY.model
    blob = synth.make_blob(m, TINY.weight_seed)
    fr = synth.render_frames(TINY.video, m.image_size, 0, TINY.n_frames)
    return m, blob, fr


# ---------------------------------------------------------------- stream compaction (exact)
def _compact_expect(masks, G):
    F, N = masks.shape
    m = masks.copy()
    m[::G] = 0
    act = m == 0
    idx = np.flatnonzero(act.reshape(-1)).astype(np.int32)
    cnt = act.sum(1)
    qoff = np.concatenate([[0], np.cumsum(cnt)]).astype(np.int32)
    pos = np.empty(F * N, np.int32)
    for f in range(F):
        r = (f // G) * G
        ranks = np.cumsum(act[f]) - 1
        for i in range(N):
            pos[f * N + i] = qoff[f] + ranks[i] if act[f, i] else qoff[r] + i
    return idx, pos, qoff


@pytest.mark.parametrize("F,N,G,p", [(8, 50, 4, 0.5), (256, 257, 8, 0.9), (128, 577, 8, 0.3),
                                     (3, 1, 2, 0.5), (2500, 3, 5, 0.6), (16, 257, 8, 1.0),
                                     (16, 257, 8, 0.0), (1, 10, 1, 0.7), (13, 300, 4, 0.5)])
def test_compact_exact(F, N, G, p):
    from paper_2506_14107_amd.dejavu import compact
    rng = np.random.default_rng(F * 1000 + N)
    masks = (rng.random((F, N)) < p).astype(np.uint8)
    masks[:, 0] = rng.integers(0, 2, F)   # the compaction does not special-case token 0
    idx, pos, qoff, cnt = compact(dev(masks), G)
    torch = require_gpu()
    torch.cuda.synchronize()
    e_idx, e_pos, e_qoff = _compact_expect(masks, G)
    c = int(host(cnt)[0])
    assert c == len(e_idx)
    assert np.array_equal(host(idx)[:c], e_idx)
    assert np.array_equal(host(qoff), e_qoff)
    assert np.array_equal(host(pos), e_pos)


# ------------------------------------------------------------ tiny fp32 model (112 px, p16, D192)
def test_tiny_gate_mode_parity():
    torch = require_gpu()
    m, blob, fr = _tiny()
    tau = float(np.float32(TINY.tau))
    enc = encoder(m, blob, 8)
    emb, masks, toks = enc.encode(dev(fr), 4, tau, want_tokens=True)
    torch.cuda.synchronize()
    mg = host(masks)
    # teacher-forced decisions: the oracle replays the GPU's map and judges every decision
    r = oracle.encode(fr, blob, m.as_dict(), 4, masks=mg)
    bad, inside = mask_parity(mg, r["cos"], tau)
    assert bad == 0, f"{bad} decisions differ outside the 1e-3 band"
    check_close(host(emb), r["emb"], "f32", "embeddings")
    check_close(host(toks), r["tokens"], "f32", "tokens")
    # untethered: the oracle's own gate
    g = oracle.encode(fr, blob, m.as_dict(), 4, tau=tau)
    agree = np.mean(g["masks"] == mg)
    assert agree > 0.99, f"gate-mode agreement {agree}"
    assert 0.1 < oracle.reuse_rate(mg, 4) < 1.0


def test_tiny_dense_matches_oracle():
    torch = require_gpu()
    m, blob, fr = _tiny()
    enc = encoder(m, blob, 8)
    emb, masks, toks = enc.encode(dev(fr), 4, float("-inf"), want_tokens=True)
    torch.cuda.synchronize()
    assert not host(masks).any()
    r = oracle.dense_vit(fr, blob, m.as_dict(), return_tokens=True)
    check_close(host(emb), r[0], "f32", "embeddings")
    check_close(host(toks), r[1], "f32", "tokens")


@pytest.mark.parametrize("m", [TINY.model, SMALL_BF16, MID_BF16, DH80_N50, N577_BF16],
                         ids=["tiny", "small", "mid", "dh80", "n577"])
def test_copy_at_plus_inf_is_bitwise(m):
    torch = require_gpu()
    blob = synth.make_blob(m, 21)
    fr = _video(m, 8, seed=3)
    enc = encoder(m, blob, 8)
    emb, masks, toks = enc.encode(dev(fr), 4, float("inf"), want_tokens=True)
    torch.cuda.synchronize()
    e, t, mk = host(emb), host(toks), host(masks)
    for f in range(8):
        r = (f // 4) * 4
        assert np.array_equal(t[f], t[r]), f"frame {f} tokens differ from reference {r}"
        assert np.array_equal(e[f], e[r])
        if f != r:
            assert mk[f, :, 1:].all() and not mk[f, :, 0].any()
    # tau = -2 is the same map reached through the gate
    emb2, masks2, toks2 = enc.encode(dev(fr), 4, -2.0, want_tokens=True)
    torch.cuda.synchronize()
    assert np.array_equal(host(masks2), mk)
    assert np.array_equal(host(toks2), t) and np.array_equal(host(emb2), e)


@pytest.mark.parametrize("m", [TINY.model, SMALL_BF16, MID_BF16, DH80_N50, N577_BF16],
                         ids=["tiny", "small", "mid", "dh80", "n577"])
def test_reuse_off_equivalences_bitwise(m):
    """tau=2 (gate runs, reuses nothing) == tau=-inf; G=1 == dense; reference frames of a
    reuse run == the same frames run densely (rows are independent of their packed slot)."""
    torch = require_gpu()
    blob = synth.make_blob(m, 22)
    fr = _video(m, 8, seed=4)
    enc = encoder(m, blob, 8)
    d_emb, _, d_tok = enc.encode(dev(fr), 4, float("-inf"), want_tokens=True)
    a_emb, a_m, a_tok = enc.encode(dev(fr), 4, 2.0, want_tokens=True)
    g_emb, _, _ = enc.encode(dev(fr), 1, 0.5)
    r_emb, r_m, _ = enc.encode(dev(fr), 4, 0.9)
    torch.cuda.synchronize()
    assert not host(a_m).any()
    assert np.array_equal(host(a_tok), host(d_tok)) and np.array_equal(host(a_emb), host(d_emb))
    assert np.array_equal(host(g_emb), host(d_emb))
    assert np.array_equal(host(r_emb)[::4], host(d_emb)[::4])
    assert not host(r_m)[::4].any() and not host(r_m)[:, :, 0].any()


def test_batching_and_determinism_bitwise():
    torch = require_gpu()
    m = SMALL_BF16
    blob = synth.make_blob(m, 23)
    fr = _video(m, 16, seed=5)
    big = encoder(m, blob, 16)
    small = encoder(m, blob, 8)
    outs = [big.encode(dev(fr), 4, 0.8, want_tokens=True) for _ in range(3)]
    o_small = small.encode(dev(fr), 4, 0.8, want_tokens=True)
    halves = [big.encode(dev(fr[:8]), 4, 0.8, want_tokens=True),
              big.encode(dev(fr[8:]), 4, 0.8, want_tokens=True)]
    torch.cuda.synchronize()
    ref = [host(t) for t in outs[0]]
    for o in outs[1:] + [o_small]:
        for a, b in zip(o, ref):
            assert np.array_equal(host(a), b)
    for k in range(3):
        cat = np.concatenate([host(halves[0][k]), host(halves[1][k])])
        assert np.array_equal(cat, ref[k])


def test_batching_bitwise_past_one_round_of_narrow_tiles():
    """Width 1152 with 257 tokens: QKV (3456 outputs), the out-projection and FC2 (1152) take the
    256 x 128 tiling, whose blocks each run one tile.  A 32-frame batch gives them well over one
    round of head tiles (QKV: 27 tile columns); the same frames encoded 8 at a time stay under one
    round.  Every output must be the same bit for bit, gated and with reuse off."""
    torch = require_gpu()
    m = ModelConfig(224, 14, 1, 1152, 18, 2304, "bf16")
    blob = synth.make_blob(m, 41)
    fr = _video(m, 32, seed=9)
    big = encoder(m, blob, 32)
    small = encoder(m, blob, 8)
    for tau in (0.9, float("-inf")):
        a = big.encode(dev(fr), 8, tau, want_tokens=True)
        b = small.encode(dev(fr), 8, tau, want_tokens=True)
        torch.cuda.synchronize()
        for x, y in zip(a, b):
            assert np.array_equal(host(x), host(y)), f"tau {tau}"


def test_live_handle_rejects_bad_arguments_without_launching():
    """A live handle rejects an empty or negative frame count, a group size of 0 or above the
    batch, a NaN tau and NULL buffers with DV_EINVAL, on the host: the output buffer keeps its
    sentinel, and the handle encodes normally afterwards."""
    torch = require_gpu()
    from paper_2506_14107_amd import dejavu as dj
    m = SMALL_BF16
    blob = synth.make_blob(m, 30)
    enc = encoder(m, blob, 8)
    fr = dev(_video(m, 8, seed=3))
    emb = torch.full((8, m.width), 7.0, dtype=torch.float32, device="cuda")
    msk = torch.zeros((8, m.depth, m.n_tokens), dtype=torch.uint8, device="cuda")
    lib, h = dj.load(), enc.handle
    s = torch.cuda.current_stream().cuda_stream
    f, e = fr.data_ptr(), emb.data_ptr()
    rcs = {
        "empty batch": lib.dv_encode(h, f, 0, 4, 0.9, e, None, s),
        "negative count": lib.dv_encode(h, f, -3, 4, 0.9, e, None, s),
        "group size 0": lib.dv_encode(h, f, 8, 0, 0.9, e, None, s),
        "group above the batch": lib.dv_encode(h, f, 8, 9, 0.9, e, None, s),
        "NaN tau": lib.dv_encode(h, f, 8, 4, float("nan"), e, None, s),
        "NULL frames": lib.dv_encode(h, None, 8, 4, 0.9, e, None, s),
        "NULL embeddings": lib.dv_encode(h, f, 8, 4, 0.9, None, None, s),
        "NULL injected maps": lib.dv_encode_masked(h, f, 8, 4, None, e, None, s),
        "empty injected batch": lib.dv_encode_masked(h, f, 0, 4, msk.data_ptr(), e, None, s),
    }
    torch.cuda.synchronize()
    bad = {k: rc for k, rc in rcs.items() if rc != dj.DV_EINVAL}
    assert not bad, f"expected DV_EINVAL: {bad}"
    assert bool(torch.all(emb == 7.0)), "a rejected call wrote the output"
    a, _, _ = enc.encode(fr, 4, 0.9)
    b, _, _ = enc.encode(fr, 4, 0.9)
    torch.cuda.synchronize()
    assert np.array_equal(host(a), host(b)) and np.isfinite(host(a)).all()


def test_mfma_probe_counts_its_work():
    """The MFMA-loop probe (measurement support) reports the FLOPs its launch performs (4 chains
    of 32x32x16 MFMAs, 32768 FLOP each, per wavefront and round), every lane writes a finite
    value to the sink, and the rate it implies is a plausible fraction of the nominal peak."""
    torch = require_gpu()
    from paper_2506_14107_amd.dejavu import dv_mfma_probe
    blocks, iters = 512, 2000
    sink = torch.full((blocks * 256,), float("nan"), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    flops = dv_mfma_probe(blocks, iters, sink.data_ptr(), stream.cuda_stream)
    assert flops == blocks * 4 * 4 * iters * 32768
    torch.cuda.synchronize()
    assert bool(torch.isfinite(sink).all())
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    dv_mfma_probe(blocks, iters, sink.data_ptr(), stream.cuda_stream)
    e.record()
    torch.cuda.synchronize()
    tflops = flops / (s.elapsed_time(e) * 1e-3) / 1e12
    assert 200 < tflops < 2600, f"{tflops:.0f} TFLOP/s"


def test_concurrent_handles_on_two_streams_bitwise():
    """Groups are independent: two handles encoding the two halves of a clip at the same time on
    two HIP streams give, bit for bit, the tokens, masks and embeddings of one encode of the whole
    clip (each handle owns its workspace; the kernels of the two streams overlap on the GPU)."""
    torch = require_gpu()
    m = N257_BF16
    blob = synth.make_blob(m, 29)
    fr = dev(_video(m, 32, seed=11, pan=0.5))
    whole = encoder(m, blob, 32)
    halves = [encoder(m, blob, 16), encoder(m, blob, 16)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    ref = [host(t) for t in whole.encode(fr, 4, 0.9, want_tokens=True)]
    for _ in range(3):
        cur = torch.cuda.current_stream()
        outs = []
        for k, (e, st) in enumerate(zip(halves, streams)):
            st.wait_stream(cur)
            with torch.cuda.stream(st):
                outs.append(e.encode(fr[16 * k:16 * (k + 1)], 4, 0.9, want_tokens=True, stream=st))
        for st in streams:
            cur.wait_stream(st)
        torch.cuda.synchronize()
        for j in range(3):
            cat = np.concatenate([host(outs[0][j]), host(outs[1][j])])
            assert np.array_equal(cat, ref[j])
    assert 0 < ref[1][4:].mean() < 1, "the clip should mix reused and recomputed tokens"


@pytest.mark.parametrize("m,n,G", [(TINY.model, 7, 4), (SMALL_BF16, 9, 4), (SMALL_BF16, 1, 4),
                                   (MID_BF16, 10, 3), (N257_BF16, 6, 4), (N577_BF16, 3, 2),
                                   (DH80_BF16, 5, 4)],
                         ids=["tiny-ragged", "small-ragged", "single-frame", "mid-G3", "n257",
                              "n577", "dh80"])
def test_injection_mode_parity(m, n, G):
    """Random, non-monotone injected maps; partial last group."""
    torch = require_gpu()
    blob = synth.make_blob(m, 24, perturb_ln=True)
    fr = _video(m, n, seed=6)
    rng = np.random.default_rng(n)
    mk = (rng.random((n, m.depth, m.n_tokens)) < 0.6).astype(np.uint8)
    enc = encoder(m, blob, 8)
    emb, eff, toks = enc.encode_masked(dev(fr), G, dev(mk), want_tokens=True)
    torch.cuda.synchronize()
    r = oracle.encode(fr, blob, m.as_dict(), G, masks=mk)
    assert np.array_equal(host(eff), r["masks"]), "effective map (class/reference forced to 0)"
    check_close(host(emb), r["emb"], m.dtype, "embeddings")
    check_close(host(toks), r["tokens"], m.dtype, "tokens")


def test_single_token_injection():
    """One reused token: its output row is the reference's; the other rows match the oracle."""
    torch = require_gpu()
    m = MID_BF16
    blob = synth.make_blob(m, 25)
    fr = _video(m, 2, seed=7)
    mk = np.zeros((2, m.depth, m.n_tokens), np.uint8)
    mk[1, m.depth - 1, 7] = 1
    enc = encoder(m, blob, 8)
    emb, _, toks = enc.encode_masked(dev(fr), 2, dev(mk), want_tokens=True)
    torch.cuda.synchronize()
    t = host(toks)
    assert np.array_equal(t[1, 7], t[0, 7])
    r = oracle.encode(fr, blob, m.as_dict(), 2, masks=mk)
    check_close(t, r["tokens"], "bf16", "tokens")


@pytest.mark.parametrize("m", [SMALL_BF16, MID_BF16, N257_BF16, DH80_BF16, W1152_BF16,
                               W1280_BF16],
                         ids=["small", "mid", "n257", "dh80", "w1152", "w1280"])
def test_bf16_gate_mode_parity(m):
    torch = require_gpu()
    blob = synth.make_blob(m, 26)
    fr = _video(m, 16, seed=8, sigma=0.02)
    enc = encoder(m, blob, 16)
    for tau in (0.6, 0.9, 0.99):
        emb, masks, toks = enc.encode(dev(fr), 8, tau, want_tokens=True)
        torch.cuda.synchronize()
        mg = host(masks)
        r = oracle.encode(fr, blob, m.as_dict(), 8, masks=mg)
        bad, inside = mask_parity(mg, r["cos"], tau)
        assert bad == 0, f"tau={tau}: {bad} decisions differ outside the band ({inside:.3%} inside)"
        assert np.all(mg[:, 1:] >= mg[:, :-1]), "gate-mode reuse must be monotone over layers"
        check_close(host(emb), r["emb"], "bf16", f"embeddings tau={tau}")
        check_close(host(toks), r["tokens"], "bf16", f"tokens tau={tau}")


# N = 577 keys in two layers: a frame's keys do not fit in LDS next to another frame's, so a
# group's frames take the per-tile wavefronts (few query tiles) or per-frame blocks
N577_L2 = ModelConfig(336, 14, 2, 128, 2, 256, "bf16")


@pytest.mark.parametrize("G,n", [(8, 21), (12, 24)], ids=["G8-ragged", "G12"])
def test_large_frame_group_gate_mode_parity(G, n):
    """Gate mode at 577 tokens over the reuse range (frames of every tile count, so both
    kernels), groups of 8 with a short last group and of 12."""
    torch = require_gpu()
    m = N577_L2
    blob = synth.make_blob(m, 27)
    fr = _video(m, n, seed=9, sigma=0.02, n_obj=4, size=40)
    enc = encoder(m, blob, 24)
    for tau in (0.5, 0.95, 0.995, 2.0):
        emb, masks, toks = enc.encode(dev(fr), G, tau, want_tokens=True)
        torch.cuda.synchronize()
        mg = host(masks)
        r = oracle.encode(fr, blob, m.as_dict(), G, masks=mg)
        bad, inside = mask_parity(mg, r["cos"], tau)
        print(f"[n577 G{G}] tau {tau}: reuse {oracle.reuse_rate(mg, G):.3f}, decisions off {bad}, "
              f"in band {inside:.2%}", flush=True)
        assert bad == 0, f"tau={tau}: {bad} decisions differ outside the band ({inside:.3%} inside)"
        check_close(host(emb), r["emb"], "bf16", f"embeddings tau={tau}")
        check_close(host(toks), r["tokens"], "bf16", f"tokens tau={tau}")
    d_emb, _, d_tok = enc.encode(dev(fr), G, float("-inf"), want_tokens=True)
    torch.cuda.synchronize()
    assert np.array_equal(host(d_tok), host(toks)), "tau = 2 equals reuse off bit for bit"
    assert np.array_equal(host(d_emb), host(emb))
