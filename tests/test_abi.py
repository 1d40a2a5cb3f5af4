"""The C ABI library on the CPU: it loads, exports every symbol the header declares,
and rejects invalid arguments on the host before any GPU work."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

from paper_2506_14107_amd import dejavu as dj

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dejavu.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*[\w\s\*]+?\b(dv_\w+)\s*\(", src, flags=re.M)))


def test_header_declares_entry_points():
    names = declared_functions()
    for n in ("dv_create", "dv_destroy", "dv_encode", "dv_encode_masked", "dv_encode_tokens",
              "dv_last_error", "dv_compact", "dv_weights_floats"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = dj.load()
    for n in declared_functions():
        assert hasattr(lib, n), f"{n} declared in dejavu.h but not exported"


def _cfg(**kw):
    base = dict(image_size=112, patch=16, depth=4, width=192, heads=3, mlp=768, dtype="f32",
                max_batch_frames=8)
    base.update(kw)
    return dj.make_config(**base)


def test_weights_floats_matches_layout():
    import synth
    w = synth.get_config("tiny").model
    assert dj.dv_weights_floats(_cfg()) == synth.weights.blob_floats(w)
    m = synth.get_config("vit_l14").model
    c = dj.make_config(m.image_size, m.patch, m.depth, m.width, m.heads, m.mlp, "bf16", 256)
    assert dj.dv_weights_floats(c) == synth.weights.blob_floats(m)
    assert dj.dv_weights_floats(_cfg(image_size=100)) == 0


def test_weights_floats_with_restoration_section():
    import dataclasses
    import synth
    m = dataclasses.replace(synth.get_config("tiny").model, restore=True)
    cfg = _cfg(flags=dj.DV_FLAG_RESTORE)
    assert dj.dv_weights_floats(cfg) == synth.weights.blob_floats(m)
    assert synth.weights.blob_floats(m) - dj.dv_weights_floats(_cfg()) == \
        m.depth * (2 * 128 * m.width + 128 + m.width)


def test_weights_floats_with_decision_section():
    import dataclasses
    import synth
    tiny = synth.get_config("tiny").model
    for restore in (False, True):
        m = dataclasses.replace(tiny, restore=restore, decision=True)
        flags = dj.DV_FLAG_DECISION | (dj.DV_FLAG_RESTORE if restore else 0)
        assert dj.dv_weights_floats(_cfg(flags=flags)) == synth.weights.blob_floats(m)
        without = dataclasses.replace(m, decision=False)
        assert synth.weights.blob_floats(m) - synth.weights.blob_floats(without) == \
            m.depth * (64 * 6 + 64 + 64 + 1)


@pytest.mark.parametrize("kw,code", [
    (dict(image_size=100), dj.DV_EUNSUPPORTED),       # S % p
    (dict(heads=5), dj.DV_EUNSUPPORTED),              # D % H
    (dict(width=96, heads=12), dj.DV_EUNSUPPORTED),   # head dim 8
    (dict(depth=0), dj.DV_EINVAL),
    (dict(max_batch_frames=0), dj.DV_EINVAL),
    (dict(dtype=7), dj.DV_EINVAL),
    (dict(width=200, heads=2), dj.DV_EUNSUPPORTED),   # width not a tile multiple
    (dict(flags=8), dj.DV_EUNSUPPORTED),              # unknown flag bit
])
def test_create_rejects_bad_config(kw, code):
    cfg = _cfg(**kw)
    w = np.zeros(16, np.float32)
    with pytest.raises(dj.DejaVuError) as e:
        dj.dv_create(cfg, w)
    assert e.value.code == code
    assert dj.dv_last_error()


def test_create_rejects_wrong_blob_size():
    cfg = _cfg()
    n = dj.dv_weights_floats(cfg)
    with pytest.raises(dj.DejaVuError) as e:
        dj.dv_create(cfg, np.zeros(n - 1, np.float32))
    assert e.value.code == dj.DV_EINVAL and "blob" in dj.dv_last_error()


def test_create_null_arguments():
    lib = dj.load()
    cfg = _cfg()
    h = ctypes.c_void_p()
    assert lib.dv_create(None, None, 0, ctypes.byref(h)) == dj.DV_EINVAL
    assert lib.dv_create(ctypes.byref(cfg), None, 0, ctypes.byref(h)) == dj.DV_EINVAL
    assert lib.dv_create(ctypes.byref(cfg), None, 0, None) == dj.DV_EINVAL


def test_encode_rejects_bad_arguments_without_a_handle():
    lib = dj.load()
    # null handle is rejected before anything touches the device
    assert lib.dv_encode(None, 1, 1, 1, 0.5, 1, None, None) == dj.DV_EINVAL
    assert lib.dv_encode_masked(None, 1, 1, 1, None, 1, None, None) == dj.DV_EINVAL
    assert lib.dv_encode_noalloc(None, 1, 1, 1, 0.5, 1, None, None) == dj.DV_EINVAL
    assert lib.dv_encode_tokens(None, 1, 1, 1, math.nan, None, 1, None, None, None) == dj.DV_EINVAL
    assert lib.dv_stream_encode(None, 1, 1, 1, 0.5, None, 1, None, None, None) == dj.DV_EINVAL
    assert lib.dv_stream_reset(None) == dj.DV_EINVAL
    held = ctypes.c_int(7)
    assert lib.dv_stream_held(None, ctypes.byref(held)) == dj.DV_EINVAL
    assert lib.dv_stream_flush(None, 1, None, None, None) == dj.DV_EINVAL
    assert lib.dv_destroy(None) == dj.DV_OK


def test_compact_rejects_bad_arguments():
    lib = dj.load()
    assert lib.dv_compact(None, 1, 1, 1, 1, 1, 1, 1, None) == dj.DV_EINVAL
    assert lib.dv_compact(1, 0, 1, 1, 1, 1, 1, 1, None) == dj.DV_EINVAL
    assert lib.dv_compact(1, 1, 1, 0, 1, 1, 1, 1, None) == dj.DV_EINVAL
    assert lib.dv_compact(1, 1 << 16, 1 << 16, 1, 1, 1, 1, 1, None) == dj.DV_EINVAL


def test_mfma_probe_rejects_bad_arguments():
    """Host validation only (no launch on error)."""
    lib = dj.load()
    fl = ctypes.c_double()
    assert lib.dv_mfma_probe(1, 1, None, ctypes.byref(fl), None) == dj.DV_EINVAL
    assert lib.dv_mfma_probe(1, 1, 1, None, None) == dj.DV_EINVAL
    assert lib.dv_mfma_probe(0, 1, 1, ctypes.byref(fl), None) == dj.DV_EINVAL
    assert lib.dv_mfma_probe(1, 0, 1, ctypes.byref(fl), None) == dj.DV_EINVAL
    assert lib.dv_mfma_probe((1 << 20) + 1, 1, 1, ctypes.byref(fl), None) == dj.DV_EINVAL


def test_profile_calls_reject_null_handle():
    lib = dj.load()
    ms, n = ctypes.c_double(), ctypes.c_longlong()
    assert lib.dv_profile(None, 1) == dj.DV_EINVAL
    assert lib.dv_profile_read(None, 0, ctypes.byref(ms), ctypes.byref(n)) == dj.DV_EINVAL
    size = ctypes.c_size_t()
    assert lib.dv_workspace_bytes(None, ctypes.byref(size)) == dj.DV_EINVAL


def test_create_reports_enomem_above_the_device_memory_cap(monkeypatch):
    """DV_MAX_DEVICE_BYTES caps a handle's device memory; the check precedes any device call, so
    it runs here without a GPU."""
    import synth
    m = synth.get_config("tiny").model
    blob = synth.make_blob(m, 1)
    monkeypatch.setenv("DV_MAX_DEVICE_BYTES", "1000")
    with pytest.raises(dj.DejaVuError) as e:
        dj.dv_create(_cfg(), blob)
    assert e.value.code == dj.DV_ENOMEM and "DV_MAX_DEVICE_BYTES" in dj.dv_last_error()


@pytest.mark.parametrize("mlp,ok,bad", [
    (4096, 2039, 2040),   # MLP hidden rows: round_up(257 B, 256) * 4096 * 2 bytes reach 2^32
    (1024, 2717, 2718),   # MLP no wider than D: the qkv rows (batch + 512 spare) * 3072 * 2 do
])
def test_config_rejects_buffers_past_32_bit_offsets(mlp, ok, bad):
    """ViT-L/14 geometry (257 tokens, width 1024, bf16): the largest batch whose every workspace
    buffer stays below 2^32 bytes is accepted, one frame more is not.  With mlp 1024 the limit
    comes from the qkv buffer and its spare rows for a stream's cached reference (2^32 / 6144 =
    699050.7 rows; 2717 frames pad to 698368 rows + 512, 2718 to 698624 + 512)."""
    def floats(b):
        return dj.dv_weights_floats(dj.make_config(224, 14, 24, 1024, 16, mlp, "bf16", b))
    assert floats(ok) > 0
    assert floats(bad) == 0
