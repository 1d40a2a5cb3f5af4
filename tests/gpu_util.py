"""Helpers for the GPU parity tests (the HIP path through the C ABI vs the CPU oracle)."""
import numpy as np

import synth
from synth.configs import ModelConfig


def require_gpu():
    import torch
    assert torch.cuda.is_available(), "these tests need the MI355X"
    return torch


def dev(a, dtype=None):
    torch = require_gpu()
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def host(t):
    return t.detach().cpu().numpy()


def encoder(m: ModelConfig, blob, max_batch_frames):
    from paper_2506_14107_amd.dejavu import Encoder
    return Encoder(m, blob, max_batch_frames)


def frame_rel_err(a, b):
    """max over frames of max_j |a_j - b_j| / max_j |b_j| (per-frame relative error)."""
    a = np.asarray(a, np.float64).reshape(len(a), -1)
    b = np.asarray(b, np.float64).reshape(len(b), -1)
    return float(np.max(np.max(np.abs(a - b), axis=1) / np.max(np.abs(b), axis=1)))


def min_cos(a, b):
    a = np.asarray(a, np.float64).reshape(len(a), -1)
    b = np.asarray(b, np.float64).reshape(len(b), -1)
    c = np.sum(a * b, 1) / (np.linalg.norm(a, axis=1) * np.linalg.norm(b, axis=1))
    return float(np.min(c))


def check_close(gpu, ref, dtype, what):
    """Output parity bar: fp32 models cos >= 0.99999 and rel <= 1e-4; bf16 cos >= 0.999 and
    rel <= 2e-2 (per frame)."""
    c, r = min_cos(gpu, ref), frame_rel_err(gpu, ref)
    cmin, rmax = (0.99999, 1e-4) if dtype == "f32" else (0.999, 2e-2)
    assert c >= cmin and r <= rmax, f"{what}: min cos {c:.6f} (>= {cmin}), rel err {r:.2e} (<= {rmax})"
    return c, r


def mask_parity(gpu_masks, oracle_cos, tau, band=1e-3):
    """Teacher-forced decision check: wherever the oracle's cosine (computed on the inputs the
    GPU's own decisions produced) is at least `band` away from tau, the GPU's decision must be
    [cos >= tau].  Returns (mismatches outside the band, fraction of evaluated tokens inside)."""
    c = np.asarray(oracle_cos)
    m = np.asarray(gpu_masks).astype(bool)
    ev = ~np.isnan(c)
    decided = ev & (np.abs(c - tau) >= band)
    bad = int(np.sum(m[decided] != (c[decided] >= tau)))
    inside = float(np.mean(np.abs(c[ev] - tau) < band)) if ev.any() else 0.0
    return bad, inside
