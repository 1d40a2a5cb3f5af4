"""Seeded random ViT weights and the flat fp32 weight blob the C ABI takes.

Blob layout (little-endian float32, tensors back to back, row-major):
    W_pe [D,3,p,p], b_pe [D], cls [D], pos [N,D]
    per layer l = 0..L-1:
        ln1_g [D], ln1_b [D], W_qkv [3D,D], b_qkv [3D], W_o [D,D], b_o [D],
        ln2_g [D], ln2_b [D], W_1 [Dm,D], b_1 [Dm], W_2 [D,Dm], b_2 [D]
    lnf_g [D], lnf_b [D]
    with the restoration MLP (ModelConfig.restore), then per layer l = 0..L-1:
        W_r1 [R,D], b_r1 [R], W_r2 [D,R], b_r2 [D]        (R = RESTORE_HIDDEN = 128)
    with the decision MLP (ModelConfig.decision), then per layer l = 0..L-1:
        W_d1 [Hd,6], b_d1 [Hd], W_d2 [1,Hd], b_d2 [1]     (Hd = DECISION_HIDDEN = 64)
Rows of W_qkv are Q, then K, then V; within each, heads are contiguous slices
of D/H rows.  Linear layers map x -> x @ W.T + b.

The restoration and decision sections come last (in that order), so the other weights of a
seed do not depend on them.
Matrices, biases, the class token and the position table are drawn from
N(0, 0.02); LayerNorm gains are 1 and shifts 0 unless ``perturb_ln`` is set,
in which case gains are 1 + N(0, 0.02) and shifts N(0, 0.02) so that the
affine part of every LayerNorm is exercised.  The decision MLP is drawn at unit scale so
that its output moves with its inputs: W_d1 and b_d1 ~ N(0, 1) except the column of the
class-token attention feature, ~ N(0, N) (that feature is about 1/N), W_d2 ~ N(0, 1/Hd),
b_d2 = 0.  For bf16 models every value is
rounded to the nearest bf16 (ties to even) and stored back as fp32, so the
blob holds exactly the weights a bf16 kernel sees.
"""
import numpy as np

from .configs import DECISION_FEATURES, DECISION_HIDDEN, RESTORE_HIDDEN, ModelConfig


def weight_layout(m: ModelConfig):
    """List of (name, shape) in blob order."""
    D, p, N, Dm = m.width, m.patch, m.n_tokens, m.mlp
    out = [("W_pe", (D, 3, p, p)), ("b_pe", (D,)), ("cls", (D,)), ("pos", (N, D))]
    for l in range(m.depth):
        out += [
            (f"l{l}.ln1_g", (D,)), (f"l{l}.ln1_b", (D,)),
            (f"l{l}.W_qkv", (3 * D, D)), (f"l{l}.b_qkv", (3 * D,)),
            (f"l{l}.W_o", (D, D)), (f"l{l}.b_o", (D,)),
            (f"l{l}.ln2_g", (D,)), (f"l{l}.ln2_b", (D,)),
            (f"l{l}.W_1", (Dm, D)), (f"l{l}.b_1", (Dm,)),
            (f"l{l}.W_2", (D, Dm)), (f"l{l}.b_2", (D,)),
        ]
    out += [("lnf_g", (D,)), ("lnf_b", (D,))]
    if m.restore:
        Rh = RESTORE_HIDDEN
        for l in range(m.depth):
            out += [(f"l{l}.W_r1", (Rh, D)), (f"l{l}.b_r1", (Rh,)),
                    (f"l{l}.W_r2", (D, Rh)), (f"l{l}.b_r2", (D,))]
    if m.decision:
        Hd, Fd = DECISION_HIDDEN, DECISION_FEATURES
        for l in range(m.depth):
            out += [(f"l{l}.W_d1", (Hd, Fd)), (f"l{l}.b_d1", (Hd,)),
                    (f"l{l}.W_d2", (1, Hd)), (f"l{l}.b_d2", (1,))]
    return out


def blob_floats(m: ModelConfig) -> int:
    return int(sum(int(np.prod(s)) for _, s in weight_layout(m)))


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), returned as float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    # finite inputs never overflow 32 bits here (only NaN patterns could)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    return r.view(np.float32).reshape(a.shape)


def make_weights(m: ModelConfig, seed: int, perturb_ln: bool = False, std: float = 0.02):
    """Dict name -> float32 array, drawn from one PCG64 stream in blob order.

    The arrays are views into one contiguous blob (``pack_weights`` of the
    returned dict equals that blob)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    blob = np.empty(blob_floats(m), dtype=np.float32)
    w, off = {}, 0
    for name, shape in weight_layout(m):
        size = int(np.prod(shape))
        v = blob[off:off + size].reshape(shape)
        off += size
        base = name.split(".")[-1]
        if base.startswith("ln") and base.endswith("_g"):
            v[...] = 1.0
            if perturb_ln:
                v += np.float32(std) * rng.standard_normal(shape, dtype=np.float32)
        elif base.startswith("ln") and base.endswith("_b"):
            v[...] = 0.0
            if perturb_ln:
                v[...] = np.float32(std) * rng.standard_normal(shape, dtype=np.float32)
        elif base in ("W_d1", "b_d1", "W_d2"):
            rng.standard_normal(shape, dtype=np.float32, out=v)
            if base == "W_d1":
                v[:, 1] *= np.float32(m.n_tokens)
            if base == "W_d2":
                v *= np.float32(1.0 / np.sqrt(shape[1]))
        elif base == "b_d2":
            v[...] = 0.0
        else:
            rng.standard_normal(shape, dtype=np.float32, out=v)
            v *= np.float32(std)
        if m.dtype == "bf16":
            v[...] = round_to_bf16(v)
        w[name] = v
    return w


def make_blob(m: ModelConfig, seed: int, perturb_ln: bool = False) -> np.ndarray:
    """The packed blob itself (what ``pack_weights(make_weights(...))`` returns), without a copy."""
    w = make_weights(m, seed, perturb_ln)
    first = w[weight_layout(m)[0][0]]
    return first.base if first.base is not None else pack_weights(w, m)


def pack_weights(w: dict, m: ModelConfig) -> np.ndarray:
    """Flatten a weight dict into the blob (1-D float32)."""
    parts = []
    for name, shape in weight_layout(m):
        a = np.asarray(w[name], dtype=np.float32)
        if a.shape != tuple(shape):
            raise ValueError(f"{name}: shape {a.shape} != {shape}")
        parts.append(a.reshape(-1))
    return np.concatenate(parts)
