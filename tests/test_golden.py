"""The oracle against what the paper states in so many words (fixtures under tests/golden/,
each naming the passage it comes from)."""
import json
import os

import oracle.reusevit as rv

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as fh:
        return json.load(fh)


def test_processing_order_follows_the_papers_pattern():
    """A group long enough for the pattern to repeat (two blocks after the I frame, G = 12):
    the frame types in processing order are the paper's I, P, B_dist2, B_dist1, B_dist1, P, ...;
    every frame comes after its references; P frames reference an earlier frame, B frames
    reference frames the stated distance away on both sides."""
    g = _load("frame_reordering.json")
    G, F = 12, 13
    order = rv.processing_order(F, G)
    n = len(g["pattern"])
    types = [rv.FRAME_TYPES[rv.reference_frames(f, G, F)[0]] for f in order[:n]]
    assert types == g["pattern"]
    seen = set()
    for f in order:
        t, past, fut = rv.reference_frames(f, G, F)
        name = rv.FRAME_TYPES[t]
        for r in (past, fut):
            if r is not None:
                assert r in seen, f"frame {f} processed before its reference {r}"
        if name == "P":
            assert past is not None and past < f and fut is None
        if name in g["reference_distance"]:
            dist = g["reference_distance"][name]
            assert past == f - dist and fut == f + dist
        seen.add(f)
    assert sorted(order) == list(range(F))


def test_patch_embedding_token_counts():
    """The oracle's patch embedding yields the token counts the paper gives for its backbones
    (patches of the image plus the class token)."""
    import numpy as np
    for b in _load("token_counts.json")["backbones"]:
        S, p, D = b["image_size"], b["patch"], 4
        N = b["tokens"]
        W = {"W_pe": np.zeros((D, 3 * p * p)), "b_pe": np.zeros(D), "cls": np.ones(D),
             "pos": np.zeros((N, D))}
        x = rv.embed(np.zeros((1, 3, S, S)), W, {"patch": p, "image_size": S, "width": D})
        assert x.shape == (1, N, D), b["name"]
        assert np.all(x[0, 0] == 1.0) and np.all(x[0, 1:] == 0.0)
