"""Per-token loop version of the reuse-aware forward, for tiny inputs (test infrastructure only).

It follows the same definition as the vectorised oracle (Section 3 of the
paper: decision by the threshold gate on the cosine similarity cue, token
filtration, recompute of C, reconstruction from the reference for R) but
walks frames, layers, tokens, heads and keys one at a time with scalar
softmax arithmetic.  It shares no helper with the vectorised oracle.  With ``cfg["restore"]``
a reused token's output adds the restoration MLP of its input difference
to the reference (hidden 128, GELU; Section 3.3), evaluated row by row.  With
``cfg["decision"]`` the gate is the decision MLP (Section 3.3): inputs the cosine, the class
token's attention weight on the token in the frame's previous layer (mean over heads; 1/N at
the first layer) and the one-hot frame type (P for every non-reference frame); reuse when its
output exceeds tau.  With ``cfg["reorder"]`` frames reference their I/P/B anchors (Section
3.1): a token compares itself with each reference, takes the larger cosine, and when reused
copies that reference (the earlier-listed, past one on a tie); a frame is computed after its
references.
"""
import math

import numpy as np


def encode_bruteforce(frames, blob, cfg, group_size, tau=None, masks=None):
    p, D, H, L, Dm = cfg["patch"], cfg["width"], cfg["heads"], cfg["depth"], cfg["mlp"]
    S = cfg["image_size"]
    gs = S // p
    N = gs * gs + 1
    dh = D // H
    flat = np.asarray(blob, dtype=np.float64).ravel()
    cur = [0]

    def nxt(*shape):
        n = int(np.prod(shape))
        a = flat[cur[0]:cur[0] + n].reshape(shape)
        cur[0] += n
        return a

    Wpe, bpe, cls, pos = nxt(D, 3 * p * p), nxt(D), nxt(D), nxt(N, D)
    layers = []
    for _ in range(L):
        layers.append([nxt(D), nxt(D), nxt(3 * D, D), nxt(3 * D), nxt(D, D), nxt(D),
                       nxt(D), nxt(D), nxt(Dm, D), nxt(Dm), nxt(D, Dm), nxt(D)])
    lnfg, lnfb = nxt(D), nxt(D)
    restore = bool(cfg.get("restore"))
    rest = [[nxt(128, D), nxt(128), nxt(D, 128), nxt(D)] for _ in range(L)] if restore else None
    decide = bool(cfg.get("decision"))
    dec = [[nxt(64, 6), nxt(64), nxt(1, 64), nxt(1)] for _ in range(L)] if decide else None

    def norm(v, gamma, beta):
        mean = sum(v) / len(v)
        var = sum((t - mean) ** 2 for t in v) / len(v)
        inv = 1.0 / math.sqrt(var + 1e-5)
        return np.array([(v[j] - mean) * inv * gamma[j] + beta[j] for j in range(len(v))])

    def cosine(a, b):
        if all(a[j] == b[j] for j in range(len(a))):
            return 1.0
        ab = sum(a[j] * b[j] for j in range(len(a)))
        aa = math.sqrt(sum(t * t for t in a))
        bb = math.sqrt(sum(t * t for t in b))
        return min(1.0, max(-1.0, ab / max(aa * bb, 1e-8)))

    F = len(frames)
    fr64 = np.asarray(frames, dtype=np.float64)
    X = np.zeros((F, N, D))
    for f in range(F):
        X[f, 0] = cls + pos[0]
        for r in range(gs):
            for c in range(gs):
                vec = fr64[f, :, r * p:(r + 1) * p, c * p:(c + 1) * p].reshape(-1)
                X[f, 1 + r * gs + c] = Wpe @ vec + bpe + pos[1 + r * gs + c]

    def decision(s, t, ftype, Wd1, bd1, Wd2, bd2):
        v = [s, t, 0.0, 0.0, 0.0, 0.0]
        v[2 + ftype] = 1.0
        out = float(bd2[0])
        for k in range(64):
            z = float(bd1[k]) + sum(float(Wd1[k, j]) * v[j] for j in range(6))
            out += float(Wd2[0, k]) * 0.5 * z * (1.0 + math.erf(z / math.sqrt(2.0)))
        return out

    reorder = bool(cfg.get("reorder"))

    def refs_of(f):
        """(type: 0 I, 1 P, 2 B_dist2, 3 B_dist1; references, past first)"""
        pos_in = f % group_size
        if not reorder:
            return (0, []) if pos_in == 0 else (1, [f - pos_in])
        if pos_in == 0:
            return 0, []
        if pos_in % 4 == 0:
            return 1, [f - 4]
        d = pos_in % 4
        base = f - d
        a, b = {1: (base, base + 2), 2: (base, base + 4), 3: (base + 2, base + 4)}[d]
        return (2 if d == 2 else 3), [a] + ([b] if b < F else [])

    M = np.zeros((F, L, N), dtype=np.uint8)
    tprev = [[1.0 / N] * N for _ in range(F)]   # class-token attention of the previous layer
    for l in range(L):
        g1, b1, Wqkv, bqkv, Wo, bo, g2, b2, W1, bb1, W2, bb2 = layers[l]
        Y = np.zeros_like(X)
        KEY = np.zeros((F, N, D))
        VAL = np.zeros((F, N, D))
        tnext = [[0.0] * N for _ in range(F)]
        done = set()

        def compute(f):
            ftype, refs = refs_of(f)
            for r in refs:                      # a frame's references are computed before it
                if r not in done:
                    compute(r)
            layer_frame(f, ftype, refs)
            done.add(f)

        def layer_frame(f, ftype, refs):
            reuse = [False] * N
            src = [f] * N
            if refs:
                for i in range(1, N):
                    sims = [cosine(X[f, i], X[r, i]) for r in refs]
                    best = 0
                    for k in range(1, len(sims)):
                        if sims[k] > sims[best]:
                            best = k
                    src[i] = refs[best]
                    if masks is not None:
                        reuse[i] = bool(masks[f][l][i])
                    elif tau == -math.inf:
                        reuse[i] = False
                    elif tau == math.inf:
                        reuse[i] = True
                    elif decide:
                        dval = decision(sims[best], tprev[f][i], ftype, *dec[l])
                        reuse[i] = dval > tau
                    else:
                        reuse[i] = sims[best] >= tau
            Q = {}
            for i in range(N):
                if reuse[i]:
                    KEY[f, i] = KEY[src[i], i]
                    VAL[f, i] = VAL[src[i], i]
                    M[f, l, i] = 2 if (reorder and src[i] != refs[0]) else 1   # 2: future
                else:
                    t = Wqkv @ norm(X[f, i], g1, b1) + bqkv
                    Q[i], KEY[f, i], VAL[f, i] = t[:D], t[D:2 * D], t[2 * D:]
            for i in range(N):
                if reuse[i]:
                    Y[f, i] = Y[src[i], i]
                    if restore:
                        Wr1, br1, Wr2, br2 = rest[l]
                        hid = Wr1 @ (X[f, i] - X[src[i], i]) + br1
                        hid = np.array([0.5 * t * (1.0 + math.erf(t / math.sqrt(2.0))) for t in hid])
                        Y[f, i] = Y[f, i] + (Wr2 @ hid + br2)
                    continue
                o = np.zeros(D)
                for h in range(H):
                    lo, hi = h * dh, (h + 1) * dh
                    sc = [float(Q[i][lo:hi] @ KEY[f, j, lo:hi]) / math.sqrt(dh) for j in range(N)]
                    mx = max(sc)
                    ex = [math.exp(s - mx) for s in sc]
                    tot = sum(ex)
                    for j in range(N):
                        o[lo:hi] += (ex[j] / tot) * VAL[f, j, lo:hi]
                        if i == 0:
                            tnext[f][j] += (ex[j] / tot) / H
                z = X[f, i] + Wo @ o + bo
                u = W1 @ norm(z, g2, b2) + bb1
                u = np.array([0.5 * t * (1.0 + math.erf(t / math.sqrt(2.0))) for t in u])
                Y[f, i] = z + W2 @ u + bb2

        for f in range(F):
            if f not in done:
                compute(f)
        X = Y
        tprev = tnext
    emb = np.stack([norm(X[f, 0], lnfg, lnfb) for f in range(F)])
    return {"emb": emb, "masks": M, "tokens": X}
