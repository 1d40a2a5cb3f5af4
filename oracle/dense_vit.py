"""A plain dense ViT forward, written separately from the reuse oracle (test infrastructure only).

It reads the weight blob with its own offset walk and computes the standard
pre-norm ViT of the paper's Section 2.3 (patchify -> linear patch embedding
-> class token + position table -> L x [LN -> MHSA -> residual, LN -> GELU
MLP -> residual] -> LayerNorm of the class token) frame by frame, with no
notion of groups or reuse.  With reuse switched off the reuse oracle must
reproduce it.
"""
import numpy as np
from scipy.special import erf


def _read_layout(blob, cfg):
    D, p, L, Dm = cfg["width"], cfg["patch"], cfg["depth"], cfg["mlp"]
    N = (cfg["image_size"] // p) ** 2 + 1
    sizes = [("W_pe", (D, 3 * p * p)), ("b_pe", (D,)), ("cls", (D,)), ("pos", (N, D))]
    for l in range(L):
        for nm, sh in (("ln1_g", (D,)), ("ln1_b", (D,)), ("W_qkv", (3 * D, D)), ("b_qkv", (3 * D,)),
                       ("W_o", (D, D)), ("b_o", (D,)), ("ln2_g", (D,)), ("ln2_b", (D,)),
                       ("W_1", (Dm, D)), ("b_1", (Dm,)), ("W_2", (D, Dm)), ("b_2", (D,))):
            sizes.append((f"{l}/{nm}", sh))
    sizes += [("lnf_g", (D,)), ("lnf_b", (D,))]
    out, pos = {}, 0
    flat = np.asarray(blob, dtype=np.float64).ravel()
    for nm, sh in sizes:
        cnt = int(np.prod(sh))
        out[nm] = flat[pos:pos + cnt].reshape(sh)
        pos += cnt
    # the restoration MLP (cfg["restore"]: W_r1 [128, D], b_r1, W_r2 [D, 128], b_r2) and then the
    # decision MLP (cfg["decision"]: W_d1 [64, 6], b_d1, W_d2 [1, 64], b_d2) may follow, one set
    # per layer; the dense forward reuses nothing, so it reads neither
    extra = L * (128 * D + 128 + D * 128 + D) if cfg.get("restore") else 0
    extra += L * (64 * 6 + 64 + 64 + 1) if cfg.get("decision") else 0
    assert pos + extra == flat.size, "weight blob size does not match the configuration"
    return out


def _ln(v, g, b, eps=1e-5):
    m = np.mean(v, axis=-1, keepdims=True)
    s2 = np.var(v, axis=-1, keepdims=True)
    return g * (v - m) / np.sqrt(s2 + eps) + b


def dense_vit(frames, blob, cfg, return_tokens=False):
    """Embeddings [F, D] (and optionally final tokens [F, N, D]) of a plain ViT."""
    p, D, H, L = cfg["patch"], cfg["width"], cfg["heads"], cfg["depth"]
    S = cfg["image_size"]
    g = S // p
    dh = D // H
    W = _read_layout(blob, cfg)
    embs, toks = [], []
    for fr in np.asarray(frames, dtype=np.float64):
        rows = [W["cls"]]
        for r in range(g):
            for c in range(g):
                patch = fr[:, r * p:(r + 1) * p, c * p:(c + 1) * p].reshape(-1)
                rows.append(W["W_pe"] @ patch + W["b_pe"])
        x = np.stack(rows) + W["pos"]
        n = x.shape[0]
        for l in range(L):
            P = lambda nm: W[f"{l}/{nm}"]  # noqa: E731
            qkv = _ln(x, P("ln1_g"), P("ln1_b")) @ P("W_qkv").T + P("b_qkv")
            q = qkv[:, :D].reshape(n, H, dh).transpose(1, 0, 2)
            k = qkv[:, D:2 * D].reshape(n, H, dh).transpose(1, 0, 2)
            v = qkv[:, 2 * D:].reshape(n, H, dh).transpose(1, 0, 2)
            a = np.einsum("hid,hjd->hij", q, k) / np.sqrt(dh)
            a = np.exp(a - a.max(axis=2, keepdims=True))
            a = a / a.sum(axis=2, keepdims=True)
            o = np.einsum("hij,hjd->hid", a, v).transpose(1, 0, 2).reshape(n, D)
            x = x + o @ P("W_o").T + P("b_o")
            u = _ln(x, P("ln2_g"), P("ln2_b")) @ P("W_1").T + P("b_1")
            u = u * 0.5 * (1.0 + erf(u / np.sqrt(2.0)))
            x = x + u @ P("W_2").T + P("b_2")
        embs.append(_ln(x[0], W["lnf_g"], W["lnf_b"]))
        toks.append(x)
    e = np.stack(embs)
    return (e, np.stack(toks)) if return_tokens else e
