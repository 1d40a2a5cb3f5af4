"""Library-routine references on the CPU (torch float64) used to pin the oracle.

The weights are loaded from the generator's named tensors, not through the
oracle's own blob reader, so a layout slip in the oracle shows up here.
"""
import numpy as np
import torch


def encoder_layer(w, l, m):
    D, H, Dm = m.width, m.heads, m.mlp
    lay = torch.nn.TransformerEncoderLayer(
        d_model=D, nhead=H, dim_feedforward=Dm, dropout=0.0, activation="gelu",
        layer_norm_eps=1e-5, batch_first=True, norm_first=True, dtype=torch.float64)
    t = lambda a: torch.tensor(np.asarray(a, dtype=np.float64))  # noqa: E731
    with torch.no_grad():
        lay.self_attn.in_proj_weight.copy_(t(w[f"l{l}.W_qkv"]))
        lay.self_attn.in_proj_bias.copy_(t(w[f"l{l}.b_qkv"]))
        lay.self_attn.out_proj.weight.copy_(t(w[f"l{l}.W_o"]))
        lay.self_attn.out_proj.bias.copy_(t(w[f"l{l}.b_o"]))
        lay.linear1.weight.copy_(t(w[f"l{l}.W_1"]))
        lay.linear1.bias.copy_(t(w[f"l{l}.b_1"]))
        lay.linear2.weight.copy_(t(w[f"l{l}.W_2"]))
        lay.linear2.bias.copy_(t(w[f"l{l}.b_2"]))
        lay.norm1.weight.copy_(t(w[f"l{l}.ln1_g"]))
        lay.norm1.bias.copy_(t(w[f"l{l}.ln1_b"]))
        lay.norm2.weight.copy_(t(w[f"l{l}.ln2_g"]))
        lay.norm2.bias.copy_(t(w[f"l{l}.ln2_b"]))
    lay.eval()
    return lay


def embed(frames, w, m):
    """conv2d patch embedding + class token + position table -> [F, N, D] float64."""
    fr = torch.tensor(np.asarray(frames, dtype=np.float64))
    Wpe = torch.tensor(np.asarray(w["W_pe"], dtype=np.float64))
    bpe = torch.tensor(np.asarray(w["b_pe"], dtype=np.float64))
    y = torch.nn.functional.conv2d(fr, Wpe, bpe, stride=m.patch)       # [F, D, g, g]
    tok = y.flatten(2).transpose(1, 2)                                   # [F, P, D]
    cls = torch.tensor(np.asarray(w["cls"], dtype=np.float64)).expand(fr.shape[0], 1, -1)
    x = torch.cat([cls, tok], dim=1)
    return x + torch.tensor(np.asarray(w["pos"], dtype=np.float64))


def vit(frames, w, m):
    """Full dense ViT from library layers: (embeddings [F, D], final tokens [F, N, D])."""
    with torch.no_grad():
        x = embed(frames, w, m)
        for l in range(m.depth):
            x = encoder_layer(w, l, m)(x)
        g = torch.tensor(np.asarray(w["lnf_g"], dtype=np.float64))
        b = torch.tensor(np.asarray(w["lnf_b"], dtype=np.float64))
        e = torch.nn.functional.layer_norm(x[:, 0], (m.width,), g, b, eps=1e-5)
    return e.numpy(), x.numpy()


def layer_with_substituted_kv(x_f, x_ref, j, w, l, m):
    """One encoder layer on frame rows x_f [N, D] whose attention keys/values at token j come
    from the reference rows x_ref instead (queries stay x_f).  K and V are linear in LN1 of
    the row, so substituting the LN1 input row substitutes the K/V row."""
    lay = encoder_layer(w, l, m)
    with torch.no_grad():
        xf = torch.tensor(np.asarray(x_f, dtype=np.float64))[None]
        xs = xf.clone()
        xs[0, j] = torch.tensor(np.asarray(x_ref[j], dtype=np.float64))
        hq, hk = lay.norm1(xf), lay.norm1(xs)
        a = lay.self_attn(hq, hk, hk, need_weights=False)[0]
        z = xf + a
        y = z + lay.linear2(torch.nn.functional.gelu(lay.linear1(lay.norm2(z))))
    return y[0].numpy()


def restoration(dx, w, l):
    """Restoration MLP of layer l (two torch Linear layers, exact erf GELU) applied to the input
    differences dx [n, D] (numpy); returns numpy float64."""
    t = lambda a: torch.tensor(np.asarray(a, dtype=np.float64))  # noqa: E731
    l1 = torch.nn.Linear(w[f"l{l}.W_r1"].shape[1], w[f"l{l}.W_r1"].shape[0], dtype=torch.float64)
    l2 = torch.nn.Linear(w[f"l{l}.W_r2"].shape[1], w[f"l{l}.W_r2"].shape[0], dtype=torch.float64)
    with torch.no_grad():
        l1.weight.copy_(t(w[f"l{l}.W_r1"]))
        l1.bias.copy_(t(w[f"l{l}.b_r1"]))
        l2.weight.copy_(t(w[f"l{l}.W_r2"]))
        l2.bias.copy_(t(w[f"l{l}.b_r2"]))
        return l2(torch.nn.functional.gelu(l1(t(dx)), approximate="none")).numpy()


def cls_attention(x_q, x_kv, w, l, m):
    """Attention weights of query 0 (the class token) over all keys in layer l, averaged over
    the heads, from torch's MultiheadAttention: queries from LN1 of the rows x_q [N, D], keys
    and values from LN1 of the rows x_kv [N, D] (numpy); returns numpy float64 [N]."""
    lay = encoder_layer(w, l, m)
    with torch.no_grad():
        hq = lay.norm1(torch.tensor(np.asarray(x_q, dtype=np.float64))[None])
        hk = lay.norm1(torch.tensor(np.asarray(x_kv, dtype=np.float64))[None])
        a = lay.self_attn(hq, hk, hk, need_weights=True, average_attn_weights=True)[1]
    return a[0, 0].numpy()


def decision_mlp(v, w, l):
    """Decision MLP of layer l (torch Linear -> exact GELU -> Linear) on features v [n, 6]
    (numpy); returns numpy float64 [n]."""
    t = lambda a: torch.tensor(np.asarray(a, dtype=np.float64))  # noqa: E731
    l1 = torch.nn.Linear(w[f"l{l}.W_d1"].shape[1], w[f"l{l}.W_d1"].shape[0], dtype=torch.float64)
    l2 = torch.nn.Linear(w[f"l{l}.W_d2"].shape[1], 1, dtype=torch.float64)
    with torch.no_grad():
        l1.weight.copy_(t(w[f"l{l}.W_d1"]))
        l1.bias.copy_(t(w[f"l{l}.b_d1"]))
        l2.weight.copy_(t(w[f"l{l}.W_d2"]))
        l2.bias.copy_(t(w[f"l{l}.b_d2"]))
        return l2(torch.nn.functional.gelu(l1(t(v)), approximate="none"))[:, 0].numpy()
