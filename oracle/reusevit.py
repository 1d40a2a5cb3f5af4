"""Vectorised CPU oracle of the reuse-aware ViT encoder forward (test infrastructure only).

What it computes, following the paper's model description (Section 3):

* ViT backbone (Section 2.3, Figure "ViT model architecture"): frames are cut
  into p x p patches, each patch is embedded linearly, a class token is added
  (placed at index 0 here) and a learned position table is added; then L
  pre-norm encoder layers (LayerNorm -> multi-head self-attention ->
  residual, LayerNorm -> 2-layer GELU MLP -> residual); the embedding is the
  final LayerNorm of the class token.
* Reference structure: frames are split into groups of G consecutive frames;
  the group's first frame is the reference and is computed in full at every
  layer (the periodic full recompute of Section 6.3, and the I-frame role of
  Section 3.1 in a star topology: every other frame of the group references
  frame 0).
* Decision (Section 3.3, similarity cue s_i of Eq. 1 with a single reference
  and the hard gate M_i = [d_i > 0] of the hard-gating equation): the learned
  MLP is replaced by the threshold d_i = cos(x_f[i], x_ref[i]) - tau with a
  ">=" tie rule, evaluated on the layer input (the residual stream before
  LayerNorm).  The class token is never reused.
* Token filtration (Section 3.3): recompute set C = {i : M_i = 0}, reuse set
  R = {i : M_i = 1}.
* Recompute on C: the whole encoder layer (QKV projection, attention,
  output projection, MLP) runs only on the rows of C.  The attention of a
  recomputed query sees all N keys/values of its frame: its own fresh K/V for
  tokens in C and the reference frame's K/V for tokens in R.
* Token reconstruction (Section 3.3): rows of C take the recomputed output,
  rows of R copy the reference frame's layer output.
* Restoration layer (Section 3.3, restoration equations), when the
  configuration enables it (``cfg["restore"]``): a reused row becomes the
  reference's layer output plus a two-layer MLP (hidden 128, GELU) of the
  difference between its own layer input and the reference's,
  y_f[i] = y_r[i] + W_r2 GELU(W_r1 (x_f[i] - x_r[i]) + b_r1) + b_r2.  The
  keys and values of reused tokens stay the reference's.  The restored rows
  are the next layer's input (so a token reused once may be recomputed later).

* Learned decision layer (Section 3.3, decision-layer equations), when the
  configuration enables it (``cfg["decision"]``): the threshold is replaced by
  d_i = MLP(v_i), v_i = (s_i, t_i, r_i) -- s_i the cosine above (one reference,
  so the max over past and future references of Eq. 1 has a single term),
  t_i the class token's attention weight on token i (mean over heads) in the
  frame's previous layer (1/N before the first layer, where no attention has
  run yet), r_i the one-hot frame type (I, P, B_dist2, B_dist1; with one
  earlier reference per group every non-reference frame is a P frame); the
  codec-metadata cue has no input here and is left out.  The MLP is two
  layers, hidden 64, exact GELU; token i is reused when d_i > tau (tau = 0
  is the paper's rule).  Such decisions are not monotone over layers, so
  every token is gated at every layer and a reused row copies the
  reference's layer output.

* Reordered referencing (Section 3.1, frame-reordering figure; Eq. 1 with two
  references), when the configuration enables it (``cfg["reorder"]``, group
  size a multiple of 4): within a group the first frame is the I frame
  (computed in full); every fourth frame after it is a P frame referencing
  the anchor four frames back; between two anchors a0 and a0 + 4 (the next
  group's I frame closing the group's last block) the middle frame is
  B_dist2, referencing both anchors, and the other two are B_dist1,
  referencing their two neighbours among a0, a0 + 2, a0 + 4.  A reference
  past the end of the call is dropped.  Frames of a layer are processed in
  the paper's order I -> (P -> B_dist2 -> B_dist1 -> B_dist1) -> ..., each
  after its references.  The similarity is the larger of the two cosines and
  a reused token takes its keys, values and layer output from the reference
  that gave it (the past one on a tie); the decision MLP's type cue is the
  frame's own type.

Modes: gate mode (``tau``) and mask-injection mode (``masks`` given; class
token and reference-frame entries are forced to 0).  ``tau = -inf`` turns
reuse off (dense), ``tau = +inf`` reuses every non-class token of every
non-reference frame; finite tau applies the literal rule.

Cosine: a.b / max(|a| |b|, 1e-8), clamped to [-1, 1], and exactly 1 when the
two rows are elementwise equal.  Arithmetic is float64 unless ``dtype`` says
otherwise.
"""
import numpy as np
from scipy.special import erf

LN_EPS = 1e-5
COS_EPS = 1e-8
RESTORE_HIDDEN = 128   # hidden width of the restoration MLP (Section 3.3)
DECISION_HIDDEN = 64   # hidden width of the decision MLP (Section 3.3 gives none)
FRAME_TYPES = ("I", "P", "B_dist2", "B_dist1")   # reference-type cue r (Section 3.3)


def unpack_blob(blob, cfg, dtype=np.float64):
    """Split the flat weight blob into named tensors (layout documented with the C ABI)."""
    D, p, L, Dm = cfg["width"], cfg["patch"], cfg["depth"], cfg["mlp"]
    N = (cfg["image_size"] // p) ** 2 + 1
    blob = np.asarray(blob)
    off = 0

    def take(*shape):
        nonlocal off
        n = int(np.prod(shape))
        if off + n > blob.size:
            raise ValueError("weight blob too short")
        a = blob[off:off + n].astype(dtype).reshape(shape)
        off += n
        return a

    W = {"W_pe": take(D, 3, p, p), "b_pe": take(D), "cls": take(D), "pos": take(N, D),
         "layers": []}
    for _ in range(L):
        lay = {}
        lay["ln1_g"], lay["ln1_b"] = take(D), take(D)
        lay["W_qkv"], lay["b_qkv"] = take(3 * D, D), take(3 * D)
        lay["W_o"], lay["b_o"] = take(D, D), take(D)
        lay["ln2_g"], lay["ln2_b"] = take(D), take(D)
        lay["W_1"], lay["b_1"] = take(Dm, D), take(Dm)
        lay["W_2"], lay["b_2"] = take(D, Dm), take(D)
        W["layers"].append(lay)
    W["lnf_g"], W["lnf_b"] = take(D), take(D)
    if cfg.get("restore"):
        R = RESTORE_HIDDEN
        for lay in W["layers"]:
            lay["W_r1"], lay["b_r1"] = take(R, D), take(R)
            lay["W_r2"], lay["b_r2"] = take(D, R), take(D)
    if cfg.get("decision"):
        Hd = DECISION_HIDDEN
        for lay in W["layers"]:
            lay["W_d1"], lay["b_d1"] = take(Hd, 2 + len(FRAME_TYPES)), take(Hd)
            lay["W_d2"], lay["b_d2"] = take(1, Hd), take(1)
    if off != blob.size:
        raise ValueError(f"weight blob has {blob.size} floats, layout needs {off}")
    return W


def layer_norm(x, g, b):
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)   # biased variance
    return (x - mu) / np.sqrt(var + LN_EPS) * g + b


def gelu(x):
    return 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))


def embed(frames, W, cfg):
    """Patch embedding + class token + position table -> x^0 [F, N, D]."""
    F = frames.shape[0]
    p = cfg["patch"]
    g = cfg["image_size"] // p
    D = cfg["width"]
    fr = np.asarray(frames, dtype=W["W_pe"].dtype)
    # patch k = (row r, col c) row-major; patch vector ordered (channel, ky, kx)
    patches = fr.reshape(F, 3, g, p, g, p).transpose(0, 2, 4, 1, 3, 5).reshape(F, g * g, 3 * p * p)
    tok = patches @ W["W_pe"].reshape(D, 3 * p * p).T + W["b_pe"]
    x = np.empty((F, g * g + 1, D), dtype=tok.dtype)
    x[:, 0] = W["cls"] + W["pos"][0]
    x[:, 1:] = tok + W["pos"][1:]
    return x


def cosine_rows(a, b):
    """Row-wise cosine similarity with the conventions stated in the module docstring."""
    dot = np.einsum("nd,nd->n", a, b)
    na = np.sqrt(np.einsum("nd,nd->n", a, a))
    nb = np.sqrt(np.einsum("nd,nd->n", b, b))
    c = np.clip(dot / np.maximum(na * nb, COS_EPS), -1.0, 1.0)
    same = np.all(a == b, axis=1)
    c[same] = 1.0
    return c


def gate_decision(cos, tau):
    """Hard gate with d_i = cos_i - tau: 1 = reuse, 0 = recompute (class token excluded by caller)."""
    if np.isnan(tau):
        raise ValueError("tau must not be NaN")
    if tau == -np.inf:
        return np.zeros(cos.shape, dtype=bool)
    if tau == np.inf:
        return np.ones(cos.shape, dtype=bool)
    return cos >= tau


def attention(q, k, v, heads, first_probs=False):
    """Multi-head softmax attention: q [n, D] against all keys k, v [N, D].  With
    ``first_probs`` also returns the attention weights of query 0 over the N keys, averaged
    over the heads."""
    n, D = q.shape
    dh = D // heads
    out = np.empty_like(q)
    p0 = np.zeros(k.shape[0], dtype=q.dtype)
    for h in range(heads):
        s = slice(h * dh, (h + 1) * dh)
        logits = (q[:, s] @ k[:, s].T) / np.sqrt(dh)
        logits -= logits.max(axis=1, keepdims=True)
        pr = np.exp(logits)
        pr /= pr.sum(axis=1, keepdims=True)
        out[:, s] = pr @ v[:, s]
        p0 += pr[0]
    return (out, p0 / heads) if first_probs else out


def reference_frames(f, group_size, n_frames):
    """(type index into FRAME_TYPES, past reference, future reference or None) of frame f under
    the reordered referencing (module docstring)."""
    G = group_size
    p = f % G
    if p == 0:
        return 0, None, None
    if p % 4 == 0:
        return 1, f - 4, None
    a0 = f - p % 4
    if p % 4 == 2:
        t, past, fut = 2, a0, a0 + 4
    elif p % 4 == 1:
        t, past, fut = 3, a0, a0 + 2
    else:
        t, past, fut = 3, a0 + 2, a0 + 4
    return t, past, (fut if fut < n_frames else None)


def processing_order(n_frames, group_size):
    """Frames of a layer in the paper's order: each group's I frame, then block by block the
    closing anchor (a P frame, or the next group's I frame), the B_dist2 frame, the two B_dist1
    frames."""
    G = group_size
    order, seen = [], set()

    def put(f):
        if f < n_frames and f not in seen:
            order.append(f)
            seen.add(f)

    for g0 in range(0, n_frames, G):
        put(g0)
        for a0 in range(g0, g0 + G, 4):
            put(a0 + 4)
            for q in (a0 + 2, a0 + 1, a0 + 3):
                if q < g0 + G:
                    put(q)
    return order


def frame_type(f, group_size):
    """Index into FRAME_TYPES: the group's first frame is the I frame, every other frame
    references it alone, the role of a P frame."""
    return 0 if f % group_size == 0 else 1


def decision_values(s, t, ftype, P):
    """d_i = MLP_decision(concat(s_i, t_i, r_i)) for one frame's tokens (Section 3.3)."""
    r = np.zeros((len(s), len(FRAME_TYPES)), dtype=P["W_d1"].dtype)
    r[:, ftype] = 1.0
    v = np.concatenate([s[:, None], t[:, None], r], axis=1)
    return (gelu(v @ P["W_d1"].T + P["b_d1"]) @ P["W_d2"].T + P["b_d2"])[:, 0]


def decision_gate(d, tau):
    """Hard gate of the decision layer: reuse when d_i > tau (the paper's rule is tau = 0);
    tau = -inf / +inf keep their meanings (reuse off / reuse everything)."""
    if np.isnan(tau):
        raise ValueError("tau must not be NaN")
    if tau == -np.inf:
        return np.zeros(d.shape, dtype=bool)
    if tau == np.inf:
        return np.ones(d.shape, dtype=bool)
    return d > tau


def qkv_rows(x_rows, P):
    D = x_rows.shape[1]
    t = layer_norm(x_rows, P["ln1_g"], P["ln1_b"]) @ P["W_qkv"].T + P["b_qkv"]
    return t[:, :D], t[:, D:2 * D], t[:, 2 * D:]


def restore_rows(dx, P):
    """Restoration MLP (Section 3.3) of the input differences dx [n, D] of reused rows."""
    return gelu(dx @ P["W_r1"].T + P["b_r1"]) @ P["W_r2"].T + P["b_r2"]


def finish_rows(x_rows, o_rows, P):
    """Output projection + residual, then the MLP sub-layer + residual."""
    z = x_rows + o_rows @ P["W_o"].T + P["b_o"]
    h = gelu(layer_norm(z, P["ln2_g"], P["ln2_b"]) @ P["W_1"].T + P["b_1"])
    return z + h @ P["W_2"].T + P["b_2"]


def reordered_layer(x, P, cfg, G, l, tau, masks, sources, t_cls, rec):
    """One layer over all frames with the reordered referencing; returns the layer output and
    the class-token attention weights of every frame (for the next layer's decision cue).
    rec: the per-(frame, layer, token) records (masks, cos, cos_past, cos_fut, src, dec, t) to
    fill.  sources (injection mode, optional): replaces the choice of reference of reused
    tokens (nonzero = the future one)."""
    F, N, D = x.shape
    H = cfg["heads"]
    decide = bool(cfg.get("decision"))
    y = np.empty_like(x)
    k_eff, v_eff = np.empty_like(x), np.empty_like(x)   # the keys/values each frame attends to
    t_next = np.empty((F, N))
    for f in processing_order(F, G):
        ftype, past, fut = reference_frames(f, G, F)
        if ftype == 0:   # I frame: the whole layer on every token
            q, k, v = qkv_rows(x[f], P)
            o, t_next[f] = attention(q, k, v, H, first_probs=True)
            y[f] = finish_rows(x[f], o, P)
            k_eff[f], v_eff[f] = k, v
            continue
        c_past = cosine_rows(x[f, 1:], x[past, 1:])
        c_fut = cosine_rows(x[f, 1:], x[fut, 1:]) if fut is not None else np.full(N - 1, -np.inf)
        s = np.maximum(c_past, c_fut)                       # similarity cue: the better reference
        from_fut = c_fut > c_past                           # a tie takes the past reference
        rec["cos"][f, l, 1:] = s
        rec["cos_past"][f, l, 1:] = c_past
        if fut is not None:
            rec["cos_fut"][f, l, 1:] = c_fut
        rec["src"][f, l, 1:] = from_fut
        if sources is not None and fut is not None:
            from_fut = np.asarray(sources[f, l, 1:]) != 0
        if decide:
            dv = decision_values(s, t_cls[f, 1:], ftype, P)
            rec["dec"][f, l, 1:] = dv
            rec["t"][f, l, 1:] = t_cls[f, 1:]
        if masks is not None:
            reuse = np.asarray(masks[f, l, 1:]) != 0
        elif decide:
            reuse = decision_gate(dv, tau)
        else:
            reuse = gate_decision(s, tau)
        m = np.concatenate([[False], reuse])                # class token never reused
        rec["masks"][f, l] = m * np.concatenate([[1], 1 + from_fut])   # 2: from the future
        C, R = np.flatnonzero(~m), np.flatnonzero(m)
        src = np.where(np.concatenate([[False], from_fut]), fut if fut is not None else past,
                       past)[R]                             # reference of each reused token
        q_c, k_c, v_c = qkv_rows(x[f, C], P)
        k_t, v_t = np.empty((N, D)), np.empty((N, D))
        k_t[C], v_t[C] = k_c, v_c                           # fresh keys/values ...
        k_t[R], v_t[R] = k_eff[src, R], v_eff[src, R]       # ... and the reference's
        o_c, t_next[f] = attention(q_c, k_t, v_t, H, first_probs=True)
        y[f, C] = finish_rows(x[f, C], o_c, P)
        y[f, R] = y[src, R]                                 # reused rows: the reference's output
        if cfg.get("restore"):
            y[f, R] += restore_rows(x[f, R] - x[src, R], P)
        k_eff[f], v_eff[f] = k_t, v_t
    return y, t_next


def encode(frames, blob, cfg, group_size, tau=None, masks=None, dtype=np.float64,
           return_layers=False, sources=None):
    """Reuse-aware encoder forward over ``frames`` [F, 3, S, S].

    Returns a dict with
      emb    [F, D]      final LayerNorm of each frame's class token
      masks  [F, L, N]   uint8, 1 = token reused at that layer
      cos    [F, L, N]   cosine to the reference token (NaN where not evaluated)
      dec    [F, L, N]   decision-MLP output d_i (only with cfg["decision"]; NaN where not
                         evaluated)
      t      [F, L, N]   its class-token attention input t_i (same conditions)
      src    [F, L, N]   with cfg["reorder"]: 1 where the future reference gave the larger
                         cosine (and supplies a reused token), 0 past, -1 not evaluated;
                         masks then hold 2 for a token reused from the future reference
      cos_past, cos_fut  [F, L, N]  the two cosines (reorder; NaN where absent)
      tokens [F, N, D]   output of the last layer
      layers (optional)  list of the L+1 token buffers x^0..x^L
    """
    if (tau is None) == (masks is None):
        raise ValueError("give exactly one of tau (gate mode) and masks (injection mode)")
    W = unpack_blob(blob, cfg, dtype)
    F = frames.shape[0]
    L, H = cfg["depth"], cfg["heads"]
    G = int(group_size)
    if F < 1 or G < 1:
        raise ValueError("need at least one frame and a group size >= 1")
    x = embed(frames, W, cfg)
    N = x.shape[1]
    out_m = np.zeros((F, L, N), dtype=np.uint8)
    out_c = np.full((F, L, N), np.nan)
    decide = bool(cfg.get("decision"))
    out_d = np.full((F, L, N), np.nan) if decide else None
    out_t = np.full((F, L, N), np.nan) if decide else None
    t_cls = np.full((F, N), 1.0 / N) if decide else None  # class-token attention, previous layer
    hist = [x.copy()] if return_layers else None
    reorder = bool(cfg.get("reorder"))
    if reorder and G % 4:
        raise ValueError("reordered referencing needs a group size that is a multiple of 4")
    out_s = np.full((F, L, N), -1, dtype=np.int8) if reorder else None
    out_cp = np.full((F, L, N), np.nan) if reorder else None
    out_cf = np.full((F, L, N), np.nan) if reorder else None

    for l in range(L):
        P = W["layers"][l]
        if reorder:
            rec = {"masks": out_m, "cos": out_c, "cos_past": out_cp, "cos_fut": out_cf,
                   "src": out_s, "dec": out_d, "t": out_t}
            x, t_cls = reordered_layer(x, P, cfg, G, l, tau, masks, sources,
                                       t_cls if decide else np.full((F, N), 1.0 / N), rec)
            if return_layers:
                hist.append(x.copy())
            continue
        y = np.empty_like(x)
        t_next = np.empty((F, N)) if decide else None
        for r in range(0, F, G):
            # reference frame: full layer on every token
            q_r, k_r, v_r = qkv_rows(x[r], P)
            o_r, p_r = attention(q_r, k_r, v_r, H, first_probs=True)
            y[r] = finish_rows(x[r], o_r, P)
            if decide:
                t_next[r] = p_r
            for f in range(r + 1, min(r + G, F)):
                c = cosine_rows(x[f, 1:], x[r, 1:])
                out_c[f, l, 1:] = c
                if decide:
                    dv = decision_values(c, t_cls[f, 1:], frame_type(f, G), P)
                    out_d[f, l, 1:] = dv
                    out_t[f, l, 1:] = t_cls[f, 1:]
                if masks is not None:
                    reuse = np.asarray(masks[f, l, 1:]) != 0
                elif decide:
                    reuse = decision_gate(dv, tau)
                else:
                    reuse = gate_decision(c, tau)
                m = np.concatenate([[False], reuse])          # class token never reused
                out_m[f, l] = m
                C = np.flatnonzero(~m)                        # recompute tokens (C[0] = class)
                q_c, k_c, v_c = qkv_rows(x[f, C], P)
                k_t, v_t = k_r.copy(), v_r.copy()             # keys/values: reference ...
                k_t[C], v_t[C] = k_c, v_c                     # ... overwritten by fresh rows
                o_c, p_c = attention(q_c, k_t, v_t, H, first_probs=True)
                y_c = finish_rows(x[f, C], o_c, P)
                if decide:
                    t_next[f] = p_c
                y[f] = y[r]                                   # reused rows: reference output
                y[f, C] = y_c                                 # recomputed rows
                if cfg.get("restore"):                        # ... calibrated by the restoration MLP
                    Rr = np.flatnonzero(m)
                    y[f, Rr] += restore_rows(x[f, Rr] - x[r, Rr], P)
        x = y
        t_cls = t_next
        if return_layers:
            hist.append(x.copy())

    emb = layer_norm(x[:, 0], W["lnf_g"], W["lnf_b"])
    res = {"emb": emb, "masks": out_m, "cos": out_c, "tokens": x}
    if decide:
        res["dec"] = out_d
        res["t"] = out_t
    if reorder:
        res["src"] = out_s
        res["cos_past"] = out_cp
        res["cos_fut"] = out_cf
    if return_layers:
        res["layers"] = hist
    return res


def reuse_rate(masks, group_size):
    """Mean of the reuse map over non-reference frames, all N tokens and all L layers
    (the reuse-rate definition of the reuse-loss equation, Section 4)."""
    F = masks.shape[0]
    nonref = [f for f in range(F) if f % group_size != 0]
    if not nonref:
        return 0.0
    return float((np.asarray(masks)[nonref] != 0).astype(np.float64).mean())
