"""Seeded synthetic video frames (stand-ins for the paper's 2 FPS evaluation clips).

Each frame is rendered independently from (recipe, frame index), so long
videos can be produced batch by batch.  A frame is:
  * a smooth periodic background: per channel
        0.5 + sum_{4 terms} a * sin(2*pi*(kx*(x + shift) + ky*y)/S + phi)
    with integer kx, ky in {1,2,3}, a ~ U(0.05, 0.15), phi ~ U(0, 2*pi);
    ``shift`` is the accumulated camera pan, which wraps seamlessly;
  * axis-aligned squares of a uniform random colour that move in a straight
    line at a fixed speed and reflect off the borders;
  * iid Gaussian pixel noise N(0, sigma) (no clipping);
then normalised as (v - 0.5) / 0.25, the harness's pixel normalisation.

A scene cut redraws background and objects from a new sub-seed.  A cyclic
motion schedule (segments) can alternate static, panning and busy spans.
"""
import numpy as np

from .configs import VideoRecipe


def _scene_of(rec: VideoRecipe, t: int):
    """(scene index, first frame of that scene)."""
    if rec.cut_first is None or t < rec.cut_first:
        return 0, 0
    k = (t - rec.cut_first) // rec.cut_every
    return 1 + k, rec.cut_first + k * rec.cut_every


def _segment_at(rec: VideoRecipe, tau: int):
    """Locate scene-local time tau in the cyclic segment schedule.

    Returns (cycle, segment index, time inside the segment, pan accumulated
    before tau)."""
    segs = rec.segments
    cyc_len = sum(s.length for s in segs)
    cyc_pan = sum(s.length * s.pan for s in segs)
    cyc, r = divmod(tau, cyc_len)
    pan = cyc * cyc_pan
    for k, s in enumerate(segs):
        if r < s.length:
            return cyc, k, r, pan + r * s.pan
        r -= s.length
        pan += s.length * s.pan
    raise AssertionError("unreachable")


def _reflect(u, lo, hi):
    span = hi - lo
    if span <= 0:
        return np.full_like(u, lo)
    m = np.mod(u - lo, 2 * span)
    return lo + np.where(m <= span, m, 2 * span - m)


def render_frame(rec: VideoRecipe, S: int, t: int) -> np.ndarray:
    """Frame t of the video, float32 [3, S, S], normalised."""
    scene, scene_start = _scene_of(rec, t)
    tau = t - scene_start
    cyc, seg_k, seg_t, shift = _segment_at(rec, tau)
    seg = rec.segments[seg_k]

    # background for this scene
    bg_rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([rec.seed, 0, scene])))
    kx = bg_rng.integers(1, 4, size=(3, 4))
    ky = bg_rng.integers(1, 4, size=(3, 4))
    amp = bg_rng.uniform(0.05, 0.15, size=(3, 4))
    phi = bg_rng.uniform(0.0, 2 * np.pi, size=(3, 4))
    ys, xs = np.meshgrid(np.arange(S, dtype=np.float64), np.arange(S, dtype=np.float64),
                         indexing="ij")
    img = np.full((3, S, S), 0.5, dtype=np.float64)
    for c in range(3):
        for j in range(4):
            img[c] += amp[c, j] * np.sin(2 * np.pi * (kx[c, j] * (xs + shift) + ky[c, j] * ys) / S
                                         + phi[c, j])

    # moving squares for this (scene, cycle, segment)
    ob_rng = np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([rec.seed, 1, scene, cyc, seg_k])))
    n, size = seg.n_objects, seg.obj_size
    colour = ob_rng.uniform(0.0, 1.0, size=(n, 3))
    start = ob_rng.uniform(0.0, S - size, size=(n, 2))
    theta = ob_rng.uniform(0.0, 2 * np.pi, size=n)
    vel = seg.speed * np.stack([np.cos(theta), np.sin(theta)], axis=1)
    posn = _reflect(start + vel * seg_t, 0.0, float(S - size))
    for o in range(n):
        x0, y0 = int(np.rint(posn[o, 0])), int(np.rint(posn[o, 1]))
        img[:, y0:y0 + size, x0:x0 + size] = colour[o][:, None, None]

    if rec.sigma > 0:
        nz_rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([rec.seed, 2, t])))
        img += rec.sigma * nz_rng.standard_normal((3, S, S))
    return ((img - 0.5) / 0.25).astype(np.float32)


def render_frames(rec: VideoRecipe, S: int, start: int, count: int) -> np.ndarray:
    """Frames [start, start+count) as float32 [count, 3, S, S]."""
    out = np.empty((count, 3, S, S), dtype=np.float32)
    for k in range(count):
        out[k] = render_frame(rec, S, start + k)
    return out
