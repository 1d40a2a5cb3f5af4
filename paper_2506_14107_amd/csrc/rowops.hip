// Row-wise kernels: patch gather, class-token init, reuse gate, stream compaction,
// LayerNorm (gathered), merge of reused rows, final LayerNorm.  All are HBM-bound;
// one 64-lane wavefront owns one row, loads are float4 and coalesced.
#include "dv_internal.h"

namespace dv {

namespace {

constexpr int WAVE = 64;
// float4 chunks of a row held per lane by the row kernels (template CK): 4 for D <= 1024, 5 for
// D <= 1280, 8 for D <= 2048

// Sum over the 64 lanes, in every lane: DPP steps within rows of 16 lanes (quad swaps, then the
// half-row and row mirrors), one LDS shuffle across rows, and the permlane32 swap across the two
// halves of the wavefront.
template <int CTRL>
__device__ inline float dpp_mov(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                                 CTRL, 0xF, 0xF, false));
}
__device__ inline float wave_sum(float v) {
    v += dpp_mov<0xB1>(v);    // quad_perm [1,0,3,2]
    v += dpp_mov<0x4E>(v);    // quad_perm [2,3,0,1]
    v += dpp_mov<0x141>(v);   // row_half_mirror
    v += dpp_mov<0x140>(v);   // row_mirror
    v += __shfl_xor(v, 16, WAVE);
    const unsigned u = __builtin_bit_cast(unsigned, v);
    const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    return v + __builtin_bit_cast(float, (threadIdx.x & 32) ? r[0] : r[1]);
}

// Buffer descriptor over `bytes` bytes at p: a load whose 32-bit byte offset falls past `bytes`
// returns zeros without a memory access (the hardware range check), so a load that is not
// needed can still be issued, which keeps the count of loads in flight the same on every path.
__device__ inline __amdgpu_buffer_rsrc_t row_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
constexpr uint32_t ROW_SKIP = 0xFFFFFFF0u;   // an offset past every row buffer (all < 2^32 bytes)

// --- patch gather: A[f*P + k, e] = frame[f][c][py*p+ky][px*p+kx], e = (c, ky, kx); zero pad to Kp
// bf16: a thread writes 8 consecutive elements of a row with one 16-byte store (Kp is a multiple
// of 64), walking (c, ky, kx) from the chunk's first element; 32-bit indices (F*P*Kp/8 < 2^31
// for every batch the handle accepts)
template <bool BF>
__global__ void im2col_k(const float* __restrict__ frames, int F, int S, int p, int Kp, void* A) {
    const int g = S / p, P = g * g, kk = 3 * p * p, pp = p * p;
    if constexpr (BF) {
        const int cpr = Kp / 8;
        const unsigned total = (unsigned)F * P * cpr;
        for (unsigned t = blockIdx.x * blockDim.x + threadIdx.x; t < total;
             t += gridDim.x * blockDim.x) {
            const unsigned row = t / cpr;
            const int e0 = (int)(t - row * cpr) * 8;
            const unsigned f = row / P;
            const int k = (int)(row - f * P);
            const int py = k / g, px = k - (k / g) * g;
            const float* base = frames + ((size_t)f * 3 * S + py * p) * S + px * p;
            int c = e0 / pp, rem = e0 - (e0 / pp) * pp;
            int ky = rem / p, kx = rem - (rem / p) * p;
            uint32_t w[4];
#pragma unroll
            for (int q = 0; q < 8; q += 2) {
                float v[2];
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    v[h] = e0 + q + h < kk ? base[((size_t)c * S + ky) * S + kx] : 0.f;
                    if (++kx == p) {
                        kx = 0;
                        if (++ky == p) {
                            ky = 0;
                            ++c;
                        }
                    }
                }
                w[q / 2] = (uint32_t)f32_to_bf16(v[0]) | ((uint32_t)f32_to_bf16(v[1]) << 16);
            }
            ((uint4*)A)[t] = uint4{w[0], w[1], w[2], w[3]};
        }
    } else {
        const size_t total = (size_t)F * P * Kp;
        for (size_t t = blockIdx.x * (size_t)blockDim.x + threadIdx.x; t < total;
             t += (size_t)gridDim.x * blockDim.x) {
            const int e = (int)(t % Kp);
            const size_t row = t / Kp;
            const int f = (int)(row / P), k = (int)(row % P);
            float v = 0.f;
            if (e < kk) {
                const int c = e / pp, ky = (e / p) % p, kx = e % p;
                const int py = k / g, px = k % g;
                v = frames[(((size_t)f * 3 + c) * S + (py * p + ky)) * S + px * p + kx];
            }
            ((float*)A)[t] = v;
        }
    }
}

__global__ void cls_init_k(float* x, const float* cls, const float* pos, int F, int N, int D) {
    const size_t total = (size_t)F * D;
    for (size_t t = blockIdx.x * (size_t)blockDim.x + threadIdx.x; t < total;
         t += (size_t)gridDim.x * blockDim.x) {
        const int f = (int)(t / D), d = (int)(t % D);
        x[(size_t)f * N * D + d] = cls[d] + pos[d];
    }
}

// --- reuse gate + LN1: blocks of GATE_TOK tokens of one frame, one wavefront per token --------
// Decides reuse for each token and, for each token that is recomputed, writes LN1 of its row
// (already in registers for the cosine) to the token-indexed buffer `ln_out`; with `d_out`
// (restoration), each reused token's difference to its reference row goes to `d_out`.
// cnt[f * chunks + block-in-frame] = number of recomputed tokens of that block.
// With `prev`, a token reused at the previous layer holds no row of its own (it is the
// reference's row): its cosine is exactly 1.  Under the decision MLP such a token may be
// recomputed; the gate then writes the reference's row into the token's row first.
// Under reordered referencing a frame has up to two references: the similarity is the larger
// cosine, `src` records which reference gave it (1: the future one; a tie keeps the past one),
// and the cosines are taken in every mode but reuse-off, since they choose the source.
template <bool BF, bool DEC, bool REORD, int CK>
__global__ __launch_bounds__(256) void gate_k(GateArgs a) {
    const int N = a.N, D = a.D;
    const int chunks = (N + GATE_TOK - 1) / GATE_TOK;
    const int f = blockIdx.x / chunks, ch = blockIdx.x % chunks;
    if (f < a.skip) {   // carried over from an earlier call: nothing to decide, no rows
        for (int i = ch * GATE_TOK + (int)threadIdx.x; i < min(N, (ch + 1) * GATE_TOK);
             i += blockDim.x)
            if (a.cur) a.cur[(size_t)f * N + i] = 0;
        if (threadIdx.x == 0 && a.cnt) a.cnt[f * chunks + ch] = 0;
        return;
    }
    // the frame's references: star -- the group's first frame (the others play P frames);
    // reordered -- its I/P/B anchors
    int ftype, r, rfut;
    if constexpr (REORD) {
        const FrameRefs q = reorder_refs(f, a.G, a.F);
        ftype = q.type;
        r = q.past;
        rfut = q.fut;
    } else {
        r = (f / a.G) * a.G;
        ftype = r == f ? 0 : 1;
        rfut = -1;
    }
    const int lane = threadIdx.x & (WAVE - 1), wave = threadIdx.x / WAVE;
    const int nwaves = blockDim.x / WAVE;
    const int nchunk = D / 4;
    __shared__ int wcount[16];
    uint8_t* om = a.out_masks ? a.out_masks + ((size_t)(f - a.skip) * a.L + a.layer) * N : nullptr;
    const float4* g4 = (const float4*)a.ln_g;
    const float4* b4 = (const float4*)a.ln_b;
    // decision MLP (Section 3.3): lane k holds hidden unit k -- its input weights for s and t,
    // its bias plus the weight of the frame's entry of the one-hot frame type, and its output
    // weight
    static_assert(DEC_HIDDEN == WAVE, "one hidden unit per lane");
    float dw_s = 0.f, dw_t = 0.f, dw_b = 0.f, dw_o = 0.f, db_o = 0.f;
    if constexpr (DEC) {
        const float* w1 = a.dec + lane * DEC_FEAT;
        dw_s = w1[0];
        dw_t = w1[1];
        dw_b = a.dec[DEC_HIDDEN * DEC_FEAT + lane] + w1[2 + ftype];
        dw_o = a.dec[DEC_HIDDEN * DEC_FEAT + DEC_HIDDEN + lane];
        db_o = a.dec[DEC_HIDDEN * DEC_FEAT + 2 * DEC_HIDDEN];
    }
    // d = w_2 . GELU(W_1 (s, t, r) + b_1) + b_2 for token i of this frame; t is the mean over
    // the heads of the class token's attention weight on i in the previous layer (1/N at the
    // first).  Every lane returns the same d.
    auto decision = [&](float cs, int i) {
        float t = 1.0f / (float)N;
        if (a.tcls) {
            float p = 0.f;
            for (int h = lane; h < a.H; h += WAVE) p += a.tcls[((size_t)f * a.H + h) * N + i];
            t = wave_sum(p) / (float)a.H;
        }
        const float z = fmaf(dw_t, t, fmaf(dw_s, cs, dw_b));
        const float g = 0.5f * z * (1.0f + erff(z * 0.70710678118654752f));
        return wave_sum(dw_o * g) + db_o;
    };
    int active = 0;
    const int i_end = min(N, (ch + 1) * GATE_TOK);
    // the previous layer's map for all of this wavefront's tokens, loaded together up front
    // (blocks of 256 threads: GATE_TOK / 4 tokens per wavefront)
    constexpr int TPW = GATE_TOK / 4;
    uint8_t pv[TPW];
    int own_k[TPW], rp_k[TPW], rq_k[TPW];   // reordered: the tokens' roots and their anchors'
#pragma unroll
    for (int k = 0; k < TPW; ++k) {
        const int i = ch * GATE_TOK + wave + k * nwaves;
        const bool in = i < i_end;
        pv[k] = (a.prev && in) ? a.prev[(size_t)f * N + i] : 0;
        own_k[k] = f;
        rp_k[k] = r;
        rq_k[k] = rfut;
        if (REORD && a.root && in && r >= 0) {
            own_k[k] = a.root[(size_t)f * N + i];
            rp_k[k] = a.root[(size_t)r * N + i];
            if (rfut >= 0) rq_k[k] = a.root[(size_t)rfut * N + i];
        }
    }
    // Cosine gate or reuse off, without restoration: the wavefront's tokens in order, the rows of
    // token kk + 1 loaded while token kk is decided and normalised (the loads of one token alone
    // leave a memory latency per token on the path).  Per token the same loads are made, or
    // skipped, and the same arithmetic in the same order as in the general loop below.
    bool fast = false;
    if constexpr (!DEC && !REORD && CK <= 5) {
        fast = (a.mode == GATE_COS || a.mode == GATE_NONE) && a.d_out == nullptr &&
               nwaves * TPW == GATE_TOK;
        if (fast) {
            const auto rx = row_rsrc(a.x, (uint32_t)((size_t)a.F * N * D * sizeof(float)));
            float4 vb[2][CK], wb[2][CK];   // the token's own row and its reference's row
            // the LN1 gain and shift in LDS: read from global memory next to a token's output,
            // their wait would also wait for the next token's rows
            __shared__ float4 sg[5 * WAVE], sb[5 * WAVE];
            for (int c = threadIdx.x; c < nchunk; c += blockDim.x) {
                sg[c] = g4[c];
                sb[c] = b4[c];
            }
            // a token reused at the previous layer has a cosine of exactly 1: its own row is read
            // only if it is recomputed all the same (tau > 1), its reference's row never
            auto fetch = [&](int kk, float4 (&vv)[CK], float4 (&ww)[CK]) {
                const int i = ch * GATE_TOK + wave + kk * nwaves;
                const bool in = i < i_end;
                const bool gated = in && a.mode == GATE_COS && ftype != 0 && i != 0;
                const bool same = gated && a.prev && pv[kk];
                const bool own = in && (!same || a.tau > 1.0f), ref = gated && !same;
                const uint32_t ob = (uint32_t)(((size_t)f * N + i) * D * sizeof(float));
                const uint32_t rb = (uint32_t)(((size_t)r * N + i) * D * sizeof(float));
#pragma unroll
                for (int k = 0; k < CK; ++k) {
                    const int c = lane + k * WAVE;
                    const bool cin = c < nchunk;
                    vv[k] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(
                        rx, (int)(own && cin ? ob + c * 16 : ROW_SKIP), 0, 0));
                    ww[k] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(
                        rx, (int)(ref && cin ? rb + c * 16 : ROW_SKIP), 0, 0));
                }
            };
            fetch(0, vb[0], wb[0]);
            __syncthreads();
#pragma unroll
            for (int kk = 0; kk < TPW; ++kk) {
                const int i = ch * GATE_TOK + wave + kk * nwaves;
                if (i >= i_end) break;
                if (kk + 1 < TPW) fetch(kk + 1, vb[(kk + 1) & 1], wb[(kk + 1) & 1]);
                const float4(&v)[CK] = vb[kk & 1];
                const float4(&w)[CK] = wb[kk & 1];
                const size_t row = (size_t)f * N + i;
                int reuse = 0;
                if (a.mode == GATE_COS && ftype != 0 && i != 0) {
                    if (a.prev && pv[kk]) {
                        reuse = a.tau <= 1.0f;
                    } else {
                        float dot = 0.f, na = 0.f, nb = 0.f;
                        int eq = 1;
#pragma unroll
                        for (int k = 0; k < CK; ++k) {
                            if (lane + k * WAVE < nchunk) {
                                const float4 u = v[k], q = w[k];
                                dot += u.x * q.x + u.y * q.y + u.z * q.z + u.w * q.w;
                                na += u.x * u.x + u.y * u.y + u.z * u.z + u.w * u.w;
                                nb += q.x * q.x + q.y * q.y + q.z * q.z + q.w * q.w;
                                eq &= (u.x == q.x) & (u.y == q.y) & (u.z == q.z) & (u.w == q.w);
                            }
                        }
                        dot = wave_sum(dot);
                        na = wave_sum(na);
                        nb = wave_sum(nb);
                        const bool same = __all(eq);
                        float cs = dot / fmaxf(sqrtf(na) * sqrtf(nb), 1e-8f);
                        cs = fminf(1.0f, fmaxf(-1.0f, cs));
                        reuse = (same ? 1.0f : cs) >= a.tau;
                    }
                }
                if (!reuse && a.ln_out) {   // as in the general loop
                    float sum = 0.f;
#pragma unroll
                    for (int k = 0; k < CK; ++k)
                        if (lane + k * WAVE < nchunk) sum += (v[k].x + v[k].y) + (v[k].z + v[k].w);
                    const float mean = wave_sum(sum) / (float)D;
                    float sq = 0.f;
#pragma unroll
                    for (int k = 0; k < CK; ++k) {
                        if (lane + k * WAVE < nchunk) {
                            const float a0 = v[k].x - mean, a1 = v[k].y - mean,
                                        a2 = v[k].z - mean, a3 = v[k].w - mean;
                            sq += (a0 * a0 + a1 * a1) + (a2 * a2 + a3 * a3);
                        }
                    }
                    const float rstd = 1.0f / sqrtf(wave_sum(sq) / (float)D + 1e-5f);
#pragma unroll
                    for (int k = 0; k < CK; ++k) {
                        const int c = lane + k * WAVE;
                        if (c < nchunk) {
                            const float4 gg = sg[c], bb = sb[c];
                            float4 o;
                            o.x = (v[k].x - mean) * rstd * gg.x + bb.x;
                            o.y = (v[k].y - mean) * rstd * gg.y + bb.y;
                            o.z = (v[k].z - mean) * rstd * gg.z + bb.z;
                            o.w = (v[k].w - mean) * rstd * gg.w + bb.w;
                            if (BF) {
                                uint2 pk;
                                pk.x = (uint32_t)f32_to_bf16(o.x) |
                                       ((uint32_t)f32_to_bf16(o.y) << 16);
                                pk.y = (uint32_t)f32_to_bf16(o.z) |
                                       ((uint32_t)f32_to_bf16(o.w) << 16);
                                ((uint2*)a.ln_out)[row * nchunk + c] = pk;
                            } else {
                                ((float4*)a.ln_out)[row * nchunk + c] = o;
                            }
                        }
                    }
                }
                if (lane == 0) {
                    if (a.cur) a.cur[row] = (uint8_t)reuse;
                    if (om) om[i] = (uint8_t)(reuse ? 1 : 0);
                    active += !reuse;
                }
            }
        }
    }
    if (!fast) {
        int k = 0;
        for (int i = ch * GATE_TOK + wave; i < i_end; i += nwaves, ++k) {
            const size_t row = (size_t)f * N + i;
            float4* xf = (float4*)(a.x + row * D);
            const float4* xo = xf;   // the token's current row (reordered: through its root)
            int reuse = 0, from_fut = 0;
            bool loaded = false;
            float4 v[CK];
            // cosine of this token's row (loaded into v on the first call) with reference row xr
            auto cosine = [&](const float4* xr) {
                float dot = 0.f, na = 0.f, nb = 0.f;
                int eq = 1;
    #pragma unroll
                for (int k = 0; k < CK; ++k) {
                    const int c = lane + k * WAVE;
                    if (c < nchunk) {
                        if (!loaded) v[k] = xo[c];
                        const float4 u = v[k], w = xr[c];
                        dot += u.x * w.x + u.y * w.y + u.z * w.z + u.w * w.w;
                        na += u.x * u.x + u.y * u.y + u.z * u.z + u.w * u.w;
                        nb += w.x * w.x + w.y * w.y + w.z * w.z + w.w * w.w;
                        eq &= (u.x == w.x) & (u.y == w.y) & (u.z == w.z) & (u.w == w.w);
                    }
                }
                loaded = true;
                dot = wave_sum(dot);
                na = wave_sum(na);
                nb = wave_sum(nb);
                const bool same = __all(eq);
                float cs = dot / fmaxf(sqrtf(na) * sqrtf(nb), 1e-8f);
                cs = fminf(1.0f, fmaxf(-1.0f, cs));
                return same ? 1.0f : cs;
            };
            if (ftype != 0 && i != 0) {
                if (a.mode == GATE_INJECT && !REORD) {
                    reuse = a.inj[((size_t)(f - a.skip) * a.L + a.layer) * N + i] != 0;
                } else if (a.mode == GATE_ALL && !REORD) {
                    reuse = 1;
                } else if (a.mode != GATE_NONE) {
                    if (a.prev && pv[k]) {
                        // a reused token stands for the reference's row: cosine exactly 1
                        if constexpr (DEC) {
                            reuse = decision(1.0f, i) > a.tau;
                            if (!reuse) {   // recomputed again: its row becomes the reference's
                                const float4* xr = (const float4*)(a.x + ((size_t)r * N + i) * D);
    #pragma unroll
                                for (int k = 0; k < CK; ++k) {
                                    const int c = lane + k * WAVE;
                                    if (c < nchunk) {
                                        v[k] = xr[c];
                                        xf[c] = v[k];
                                    }
                                }
                                loaded = true;
                            }
                        } else {
                            reuse = a.tau <= 1.0f;
                        }
                    } else {
                        // reordered: rows are read through the previous layer's roots (a token reused
                        // there is the row of the frame that recomputed it); one root, one row, and
                        // a cosine of exactly 1 without reading it
                        const int own = own_k[k], rp = rp_k[k], rq = rq_k[k];
                        if (REORD && a.root) xo = (const float4*)(a.x + ((size_t)own * N + i) * D);
                        float cs = own == rp ? 1.0f
                                             : cosine((const float4*)(a.x + ((size_t)rp * N + i) * D));
                        // the better of the two references; a past cosine of exactly 1 (the same
                        // root) already wins, a tie going to the past one, so the future one is
                        // not needed
                        if (REORD && rfut >= 0 && own != rp) {
                            const float c2 =
                                own == rq ? 1.0f
                                          : cosine((const float4*)(a.x + ((size_t)rq * N + i) * D));
                            from_fut = c2 > cs;
                            cs = fmaxf(cs, c2);
                        }
                        if (a.mode == GATE_INJECT) {
                            reuse = a.inj[((size_t)(f - a.skip) * a.L + a.layer) * N + i] != 0;
                        } else if (a.mode == GATE_ALL) {
                            reuse = 1;
                        } else if constexpr (DEC) {
                            reuse = decision(cs, i) > a.tau;
                        } else {
                            reuse = cs >= a.tau;
                        }
                        if (REORD && !reuse && own != f) {   // recomputed after being reused: the
    #pragma unroll                                           // token gets its root's row back
                            for (int k = 0; k < CK; ++k) {
                                const int c = lane + k * WAVE;
                                if (c < nchunk) {
                                    if (!loaded) v[k] = xo[c];
                                    xf[c] = v[k];
                                }
                            }
                            loaded = true;
                        }
                    }
                }
            }
            if (reuse && a.d_out) {   // reused (restoration): x_f - x_ref into the token-indexed buffer
                const int rs = from_fut ? rfut : r;   // the reference that supplies the token
                const float4* xr = (const float4*)(a.x + ((size_t)rs * N + i) * D);
    #pragma unroll
                for (int k = 0; k < CK; ++k) {
                    const int c = lane + k * WAVE;
                    if (c < nchunk) {
                        const float4 u = loaded ? v[k] : xf[c], w = xr[c];
                        const float4 o = {u.x - w.x, u.y - w.y, u.z - w.z, u.w - w.w};
                        if (BF) {
                            uint2 pk;
                            pk.x = (uint32_t)f32_to_bf16(o.x) | ((uint32_t)f32_to_bf16(o.y) << 16);
                            pk.y = (uint32_t)f32_to_bf16(o.z) | ((uint32_t)f32_to_bf16(o.w) << 16);
                            ((uint2*)a.d_out)[row * nchunk + c] = pk;
                        } else {
                            ((float4*)a.d_out)[row * nchunk + c] = o;
                        }
                    }
                }
            }
            if (!reuse && a.ln_out) {   // recomputed: LN1 of the row into the token-indexed buffer
                if (!loaded) {
    #pragma unroll
                    for (int k = 0; k < CK; ++k) {
                        const int c = lane + k * WAVE;
                        if (c < nchunk) v[k] = xo[c];
                    }
                }
                float sum = 0.f;
    #pragma unroll
                for (int k = 0; k < CK; ++k)
                    if (lane + k * WAVE < nchunk) sum += (v[k].x + v[k].y) + (v[k].z + v[k].w);
                const float mean = wave_sum(sum) / (float)D;
                float sq = 0.f;
    #pragma unroll
                for (int k = 0; k < CK; ++k) {
                    if (lane + k * WAVE < nchunk) {
                        const float a0 = v[k].x - mean, a1 = v[k].y - mean, a2 = v[k].z - mean,
                                    a3 = v[k].w - mean;
                        sq += (a0 * a0 + a1 * a1) + (a2 * a2 + a3 * a3);
                    }
                }
                const float rstd = 1.0f / sqrtf(wave_sum(sq) / (float)D + 1e-5f);
    #pragma unroll
                for (int k = 0; k < CK; ++k) {
                    const int c = lane + k * WAVE;
                    if (c < nchunk) {
                        const float4 gg = g4[c], bb = b4[c];
                        float4 o;
                        o.x = (v[k].x - mean) * rstd * gg.x + bb.x;
                        o.y = (v[k].y - mean) * rstd * gg.y + bb.y;
                        o.z = (v[k].z - mean) * rstd * gg.z + bb.z;
                        o.w = (v[k].w - mean) * rstd * gg.w + bb.w;
                        if (BF) {
                            uint2 pk;
                            pk.x = (uint32_t)f32_to_bf16(o.x) | ((uint32_t)f32_to_bf16(o.y) << 16);
                            pk.y = (uint32_t)f32_to_bf16(o.z) | ((uint32_t)f32_to_bf16(o.w) << 16);
                            ((uint2*)a.ln_out)[row * nchunk + c] = pk;
                        } else {
                            ((float4*)a.ln_out)[row * nchunk + c] = o;
                        }
                    }
                }
            }
            if (lane == 0) {
                if (a.cur) a.cur[row] = (uint8_t)reuse;
                if (REORD) a.src[row] = (uint8_t)from_fut;
                if (om) om[i] = (uint8_t)(reuse ? 1 + from_fut : 0);   // 2: from the future anchor
                active += !reuse;
            }
        }
    }
    if (lane == 0) wcount[wave] = active;
    __syncthreads();
    if (threadIdx.x == 0 && a.cnt) {
        int s = 0;
        for (int w = 0; w < nwaves; ++w) s += wcount[w];
        a.cnt[f * chunks + ch] = s;
    }
}

__global__ __launch_bounds__(256) void count_k(const uint8_t* m, int F, int N, int G, int* cnt) {
    const int f = blockIdx.x;
    const bool ref = (f % G) == 0;
    int c = 0;
    for (int i = threadIdx.x; i < N; i += blockDim.x) c += ref || m[(size_t)f * N + i] == 0;
    __shared__ int red[256];
    red[threadIdx.x] = c;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if ((int)threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
        __syncthreads();
    }
    if (threadIdx.x == 0) cnt[f] = red[0];
}

// --- exclusive prefix over frames: qoff[f] = sum_{g<f} count(g), qoff[F] = M[0] = total ------
// count(g) = cnt[g*per] + ... + cnt[g*per + per-1]; one block; qoff may equal cnt when per == 1
// (each thread reads its entries before any write to them)
__global__ __launch_bounds__(1024) void scan_k(const int* cnt, int per, int F, int tokens, int* qoff,
                                              int* M) {
    __shared__ int part[1024];
    __shared__ int carry_s;
    const int tid = threadIdx.x;
    if (tid == 0) carry_s = 0;
    __syncthreads();
    for (int base = 0; base < F; base += 1024) {
        const int f = base + tid;
        int v = 0;
        if (f < F)
            for (int k = 0; k < per; ++k) v += cnt[(size_t)f * per + k];
        part[tid] = v;
        __syncthreads();
        for (int o = 1; o < 1024; o <<= 1) {  // Hillis-Steele inclusive scan
            const int add = tid >= o ? part[tid - o] : 0;
            __syncthreads();
            part[tid] += add;
            __syncthreads();
        }
        const int carry = carry_s;
        if (f < F) qoff[f] = carry + part[tid] - v;
        __syncthreads();
        if (tid == 1023) carry_s = carry + part[1023];
        __syncthreads();
    }
    if (tid == 0) {
        qoff[F] = carry_s;
        M[0] = carry_s;
        if (tokens > 0) M[1] = tokens - carry_s;   // reused tokens
    }
}

// --- stream compaction: one block (256 threads) per frame ------------------------------------
// Frame f's recomputed tokens go to packed slots qoff[f] .. qoff[f+1] in token order; the rank
// inside the frame comes from a wavefront ballot + popcount and a prefix over the block's four
// wavefronts.  A reused token points at the slot of the same token of its reference frame
// (reference frames keep all their tokens, in order).  cur == nullptr: every token recomputed,
// qoff ignored (identity lists).  ridx: the complement list of reused tokens, frame-major (a
// reused token's rank is i minus the recomputed tokens of its frame before i).
// With `cnt` (the gate's per-block counts, `per` of them per frame) the frame offsets come from
// the counts themselves: each block sums the counts of the frames before it (and before its
// reference) and writes qoff[f]; the last block writes qoff[F], M[0] = the recomputed rows and,
// with tokens > 0, M[1] = tokens - M[0].  The offsets equal those of scan_k.
__global__ __launch_bounds__(256) void compact_k(const uint8_t* cur, const int* qoff_in, int F,
                                                 int N, int G, int* idx, int* pos, int* qoff_out,
                                                 int* ridx, int skip, int ext_row, int* rslot,
                                                 const int* cnt, int per, int* qoff_w, int* M,
                                                 int tokens) {
    const int f = blockIdx.x;
    const int r = (f / G) * G;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    __shared__ int wtot[4];
    int pre_f = 0, pre_r = 0;   // counts of the frames before f and before r
    if (cnt) {
        // eight independent loads per thread per pass: the last frames' blocks sum thousands of
        // counts, and one load in flight per pass would put a memory latency per 256 of them on
        // the kernel's critical path.  a: frames before f, b: before r, c: up to lim (the last
        // block also takes its own frame's counts, for the total)
        constexpr int U = 8;
        const int lim = (f == F - 1 ? f + 1 : f) * per;
        int a = 0, b = 0, c = 0;
        for (int e0 = 0; e0 < lim; e0 += 256 * U) {
            int v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int e = e0 + u * 256 + tid;
                v[u] = e < lim ? cnt[e] : 0;
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int e = e0 + u * 256 + tid;
                a += e < f * per ? v[u] : 0;
                b += e < r * per ? v[u] : 0;
                c += v[u];
            }
        }
        for (int o = 32; o >= 1; o >>= 1) {
            a += __shfl_xor(a, o, WAVE);
            b += __shfl_xor(b, o, WAVE);
            c += __shfl_xor(c, o, WAVE);
        }
        __shared__ int wsum3[3][4];
        if (lane == 0) {
            wsum3[0][wave] = a;
            wsum3[1][wave] = b;
            wsum3[2][wave] = c;
        }
        __syncthreads();
        pre_f = wsum3[0][0] + wsum3[0][1] + wsum3[0][2] + wsum3[0][3];
        pre_r = wsum3[1][0] + wsum3[1][1] + wsum3[1][2] + wsum3[1][3];
        if (tid == 0) {
            qoff_w[f] = pre_f;
            if (f == F - 1) {
                const int total = wsum3[2][0] + wsum3[2][1] + wsum3[2][2] + wsum3[2][3];
                qoff_w[F] = total;
                M[0] = total;
                if (tokens > 0) M[1] = tokens - total;
            }
        }
    }
    if (f < skip) {   // carried over from an earlier call: no rows; the cached reference's
                      // keys/values are the rows at ext_row (the other such frames are never read)
        for (int i = tid; i < N; i += 256) pos[(size_t)f * N + i] = ext_row + i;
        return;
    }
    const int off = cnt ? pre_f : cur ? qoff_in[f] : f * N;
    const int refoff = (skip > 0 && r == 0) ? ext_row : cnt ? pre_r : cur ? qoff_in[r] : r * N;
    int running = 0;
    for (int base = 0; base < N; base += 256) {
        const int i = base + tid;
        const bool valid = i < N;
        const bool act = valid && (cur == nullptr || f == r || cur[(size_t)f * N + i] == 0);
        const unsigned long long bal = __ballot(act);
        const int lpre = __popcll(bal & ((1ull << lane) - 1ull));
        __syncthreads();  // previous chunk's wtot reads are done
        if (lane == 0) wtot[wave] = __popcll(bal);
        __syncthreads();
        int wpre = 0;
        for (int w = 0; w < wave; ++w) wpre += wtot[w];
        const int rank = running + wpre + lpre;
        if (act) {
            idx[off + rank] = f * N + i;
            pos[(size_t)f * N + i] = off + rank;
        } else if (valid) {
            pos[(size_t)f * N + i] = refoff + i;
            // rank among reused tokens: those of earlier frames, then the frame's before i
            const int slot = ((f - skip) * N - off) + i - rank;
            if (ridx) ridx[slot] = f * N + i;
            if (rslot) rslot[(size_t)f * N + i] = slot;
        }
        running += wtot[0] + wtot[1] + wtot[2] + wtot[3];
    }
    if (!cur && tid == 0) {
        qoff_out[f] = off;
        if (f == F - 1) qoff_out[F] = F * N;
    }
}

// --- LayerNorm of (gathered) rows -> elem rows ------------------------------------------------
template <bool BF, int CK>
__global__ __launch_bounds__(256) void ln_rows_k(const float* __restrict__ src,
                                                 const int* __restrict__ gather,
                                                 const int* __restrict__ Mdev, int Mmax, int D,
                                                 const float* __restrict__ g,
                                                 const float* __restrict__ b, void* dst) {
    const int M = Mdev ? *Mdev : Mmax;
    const int lane = threadIdx.x & 63;
    const int nchunk = D / 4;
    const float4* g4 = (const float4*)g;
    const float4* b4 = (const float4*)b;
    for (int row = (blockIdx.x * blockDim.x + threadIdx.x) / 64; row < M;
         row += gridDim.x * blockDim.x / 64) {
        const int srow = gather ? gather[row] : row;
        const float4* s4 = (const float4*)(src + (size_t)srow * D);
        float4 v[CK];
        float sum = 0.f;
#pragma unroll
        for (int k = 0; k < CK; ++k) {
            const int c = lane + k * 64;
            if (c < nchunk) {
                v[k] = s4[c];
                sum += (v[k].x + v[k].y) + (v[k].z + v[k].w);
            }
        }
        const float mean = wave_sum(sum) / (float)D;
        float sq = 0.f;
#pragma unroll
        for (int k = 0; k < CK; ++k) {
            const int c = lane + k * 64;
            if (c < nchunk) {
                const float a0 = v[k].x - mean, a1 = v[k].y - mean, a2 = v[k].z - mean,
                            a3 = v[k].w - mean;
                sq += (a0 * a0 + a1 * a1) + (a2 * a2 + a3 * a3);
            }
        }
        const float rstd = 1.0f / sqrtf(wave_sum(sq) / (float)D + 1e-5f);
#pragma unroll
        for (int k = 0; k < CK; ++k) {
            const int c = lane + k * 64;
            if (c < nchunk) {
                const float4 gg = g4[c], bb = b4[c];
                float4 o;
                o.x = (v[k].x - mean) * rstd * gg.x + bb.x;
                o.y = (v[k].y - mean) * rstd * gg.y + bb.y;
                o.z = (v[k].z - mean) * rstd * gg.z + bb.z;
                o.w = (v[k].w - mean) * rstd * gg.w + bb.w;
                if (BF) {
                    uint2 pk;
                    pk.x = (uint32_t)f32_to_bf16(o.x) | ((uint32_t)f32_to_bf16(o.y) << 16);
                    pk.y = (uint32_t)f32_to_bf16(o.z) | ((uint32_t)f32_to_bf16(o.w) << 16);
                    ((uint2*)dst)[(size_t)row * nchunk + c] = pk;
                } else {
                    ((float4*)dst)[(size_t)row * nchunk + c] = o;
                }
            }
        }
    }
}

__global__ __launch_bounds__(256) void merge_k(float* x, const uint8_t* cur, const int* root, int F,
                                               int N, int D, int G) {
    const int lane = threadIdx.x & 63;
    const int total = F * N;
    for (int t = (blockIdx.x * blockDim.x + threadIdx.x) / 64; t < total;
         t += gridDim.x * blockDim.x / 64) {
        if (!cur[t]) continue;
        const int f = t / N, i = t % N;
        const int r = root ? root[t] : (f / G) * G;
        if (r == f) continue;
        const float4* s = (const float4*)(x + ((size_t)r * N + i) * D);
        float4* d = (float4*)(x + (size_t)t * D);
        for (int c = lane; c < D / 4; c += 64) d[c] = s[c];
    }
}

// --- reordered referencing: where a reused token's key/value row and new row come from -------
// A reused token takes them from the same token of the reference that supplied it, which may be
// reused in turn; the chain ends at a frame that recomputes the token (I frames recompute every
// token, and every step moves to an earlier frame of the processing order, so a chain is at
// most a few frames long).  pos of recomputed tokens is already set; reused ones copy it.
// root: for every token, the frame whose row after this layer is the token's next row.
__global__ __launch_bounds__(256) void resolve_k(const uint8_t* __restrict__ cur,
                                                 const uint8_t* __restrict__ src, int F, int N,
                                                 int G, int* pos, int* root) {
    const int total = F * N;
    for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < total; t += gridDim.x * blockDim.x) {
        if (!cur[t]) {   // recomputed: its own frame holds its next row
            root[t] = t / N;
            continue;
        }
        const int i = t % N;
        int r = t / N;
        for (int hop = 0; hop < 64 && cur[(size_t)r * N + i]; ++hop) {
            const FrameRefs q = reorder_refs(r, G, F);
            const int next = src[(size_t)r * N + i] ? q.fut : q.past;
            if (next < 0) break;
            r = next;
        }
        pos[t] = pos[(size_t)r * N + i];
        root[t] = r;
    }
}

// --- keys/values of frame f (token i's at packed row pos[f*N + i]: its own, or its source's
// when reused) to a dense [N, 2D] copy: the reference carried to the next call of a stream
__global__ __launch_bounds__(256) void copy_ref_kv_k(const void* qkv, const int* pos, int f, int N,
                                                     int D, int el, void* dst) {
    const size_t per = (size_t)2 * D * el / 16;   // 16-byte pieces of a key/value row
    const size_t total = (size_t)N * per;
    for (size_t t = blockIdx.x * (size_t)blockDim.x + threadIdx.x; t < total;
         t += (size_t)gridDim.x * blockDim.x) {
        const size_t i = t / per, c = t % per;
        const size_t row = (size_t)pos[(size_t)f * N + i];
        const uint4* src = (const uint4*)((const char*)qkv + (row * 3 * D + D) * el);
        ((uint4*)dst)[t] = src[c];
    }
}

// --- frame f's token rows to a dense [N, D] copy; with `root`, token i's row is that of frame
// root[f*N + i] (reordered referencing: reused rows are aliases of the frame recomputing them)
__global__ __launch_bounds__(256) void copy_rows_k(const float* x, const int* root, int f, int N,
                                                   int D, float* dst) {
    const int lane = threadIdx.x & 63;
    for (int i = (blockIdx.x * blockDim.x + threadIdx.x) / 64; i < N;
         i += gridDim.x * blockDim.x / 64) {
        const int r = root ? root[(size_t)f * N + i] : f;
        const float4* s = (const float4*)(x + ((size_t)r * N + i) * D);
        float4* d = (float4*)(dst + (size_t)i * D);
        for (int c = lane; c < D / 4; c += 64) d[c] = s[c];
    }
}

// --- reordered referencing with the restoration layer: one wavefront per reused token --------
// Its new row is its source token's new row plus its own restoration output; the source may be
// reused in turn, so the row is built from the chain's root (a frame recomputing the token, whose
// new row FC2 wrote) outward, adding each link's restoration output, the token's own last.
__global__ __launch_bounds__(256) void restore_chain_k(float* x, const float* __restrict__ rbuf,
                                                       const int* __restrict__ ridx,
                                                       const int* __restrict__ rslot,
                                                       const uint8_t* __restrict__ cur,
                                                       const uint8_t* __restrict__ src,
                                                       const int* Mdev, int F, int N, int D,
                                                       int G) {
    const int lane = threadIdx.x & 63;
    const int M = *Mdev;
    for (int r = (blockIdx.x * blockDim.x + threadIdx.x) / 64; r < M;
         r += gridDim.x * blockDim.x / 64) {
        const int t = ridx[r], i = t % N;
        int link[CHAIN_MAX];   // the chain's reused tokens' frames, the token's own first
        int n = 0, g = t / N;
        while (n < CHAIN_MAX && cur[(size_t)g * N + i]) {
            link[n++] = g;
            const FrameRefs q = reorder_refs(g, G, F);
            const int next = src[(size_t)g * N + i] ? q.fut : q.past;
            if (next < 0) break;
            g = next;
        }
        const float4* root = (const float4*)(x + ((size_t)g * N + i) * D);
        float4* out = (float4*)(x + (size_t)t * D);
        for (int c = lane; c < D / 4; c += 64) {
            float4 v = root[c];
            for (int k = n - 1; k >= 0; --k) {
                const size_t slot = (size_t)rslot[(size_t)link[k] * N + i];
                const float4 d = ((const float4*)(rbuf + slot * D))[c];
                v.x += d.x;
                v.y += d.y;
                v.z += d.z;
                v.w += d.w;
            }
            out[c] = v;
        }
    }
}

__global__ __launch_bounds__(256) void final_ln_k(const float* x, int F, int N, int D,
                                                  const float* g, const float* b, float* emb) {
    const int lane = threadIdx.x & 63;
    for (int f = (blockIdx.x * blockDim.x + threadIdx.x) / 64; f < F;
         f += gridDim.x * blockDim.x / 64) {
        const float* row = x + (size_t)f * N * D;
        float s = 0.f;
        for (int d = lane; d < D; d += 64) s += row[d];
        const float mean = wave_sum(s) / (float)D;
        float q = 0.f;
        for (int d = lane; d < D; d += 64) {
            const float a = row[d] - mean;
            q += a * a;
        }
        const float rstd = 1.0f / sqrtf(wave_sum(q) / (float)D + 1e-5f);
        for (int d = lane; d < D; d += 64) emb[(size_t)f * D + d] = (row[d] - mean) * rstd * g[d] + b[d];
    }
}

__global__ void fill_u8_k(uint8_t* p, size_t n, uint8_t v) {
    for (size_t t = blockIdx.x * (size_t)blockDim.x + threadIdx.x; t < n;
         t += (size_t)gridDim.x * blockDim.x)
        p[t] = v;
}

__global__ void zero_mask_layer_k(uint8_t* om, int F, int L, int N, int layer) {
    const size_t total = (size_t)F * N;
    for (size_t t = blockIdx.x * (size_t)blockDim.x + threadIdx.x; t < total;
         t += (size_t)gridDim.x * blockDim.x) {
        const size_t f = t / N, i = t % N;
        om[(f * L + layer) * N + i] = 0;
    }
}

inline int grid_for(size_t work, int per_block, int cap = 8192) {
    size_t g = (work + per_block - 1) / per_block;
    if (g < 1) g = 1;
    return (int)(g < (size_t)cap ? g : (size_t)cap);
}

}  // namespace

void launch_im2col(bool bf16, const float* frames, int F, int S, int p, int Kp, void* A,
                   hipStream_t s) {
    const int P = (S / p) * (S / p);
    const size_t total = (size_t)F * P * Kp / (bf16 ? 8 : 1);   // elements, or 8-element chunks
    const int grid = grid_for(total, 256, 65536);
    if (bf16) hipLaunchKernelGGL(im2col_k<true>, dim3(grid), dim3(256), 0, s, frames, F, S, p, Kp, A);
    else hipLaunchKernelGGL(im2col_k<false>, dim3(grid), dim3(256), 0, s, frames, F, S, p, Kp, A);
}

void launch_cls_init(float* x, const float* cls, const float* pos, int F, int N, int D,
                     hipStream_t s) {
    hipLaunchKernelGGL(cls_init_k, dim3(grid_for((size_t)F * D, 256)), dim3(256), 0, s, x, cls,
                       pos, F, N, D);
}

template <int CK>
void launch_gate_ck(int v, dim3 grid, dim3 block, const GateArgs& a, hipStream_t s) {
    switch (v) {
        case 0: hipLaunchKernelGGL((gate_k<false, false, false, CK>), grid, block, 0, s, a); break;
        case 1: hipLaunchKernelGGL((gate_k<false, false, true, CK>), grid, block, 0, s, a); break;
        case 2: hipLaunchKernelGGL((gate_k<false, true, false, CK>), grid, block, 0, s, a); break;
        case 3: hipLaunchKernelGGL((gate_k<false, true, true, CK>), grid, block, 0, s, a); break;
        case 4: hipLaunchKernelGGL((gate_k<true, false, false, CK>), grid, block, 0, s, a); break;
        case 5: hipLaunchKernelGGL((gate_k<true, false, true, CK>), grid, block, 0, s, a); break;
        case 6: hipLaunchKernelGGL((gate_k<true, true, false, CK>), grid, block, 0, s, a); break;
        default: hipLaunchKernelGGL((gate_k<true, true, true, CK>), grid, block, 0, s, a); break;
    }
}

void launch_gate(bool bf16, const GateArgs& a, hipStream_t s) {
    const dim3 grid(a.F * gate_chunks(a.N)), block(256);
    const bool dec = a.dec != nullptr && a.mode == GATE_COS;
    const int v = (bf16 ? 4 : 0) + (dec ? 2 : 0) + (a.reorder ? 1 : 0);
    // as few float4 chunks per lane as the row needs: fewer registers, more waves per SIMD
    if (a.D <= 1024) launch_gate_ck<4>(v, grid, block, a, s);
    else if (a.D <= 1280) launch_gate_ck<5>(v, grid, block, a, s);
    else launch_gate_ck<8>(v, grid, block, a, s);
}

void launch_count(const uint8_t* m, int F, int N, int G, int* cnt, hipStream_t s) {
    hipLaunchKernelGGL(count_k, dim3(F), dim3(256), 0, s, m, F, N, G, cnt);
}

void launch_scan(const int* cnt, int per, int F, int tokens, int* qoff, int* M, hipStream_t s) {
    hipLaunchKernelGGL(scan_k, dim3(1), dim3(1024), 0, s, cnt, per, F, tokens, qoff, M);
}

void launch_compact(const uint8_t* cur, const int* qoff_in, int F, int N, int G, int* idx,
                    int* pos, int* qoff_out, int* ridx, hipStream_t s, int skip, int ext_row,
                    int* rslot) {
    hipLaunchKernelGGL(compact_k, dim3(F), dim3(256), 0, s, cur, qoff_in, F, N, G, idx, pos,
                       qoff_out, ridx, skip, ext_row, rslot, nullptr, 0, nullptr, nullptr, 0);
}

void launch_scan_compact(const int* cnt, int per, int tokens, const uint8_t* cur, int F, int N,
                         int G, int* idx, int* pos, int* qoff, int* M, int* ridx, hipStream_t s,
                         int skip, int ext_row, int* rslot) {
    hipLaunchKernelGGL(compact_k, dim3(F), dim3(256), 0, s, cur, nullptr, F, N, G, idx, pos,
                       nullptr, ridx, skip, ext_row, rslot, cnt, per, qoff, M, tokens);
}

void launch_restore_chain(float* x, const float* rbuf, const int* ridx, const int* rslot,
                          const uint8_t* cur, const uint8_t* src, const int* Mdev, int Mmax, int F,
                          int N, int D, int G, hipStream_t s) {
    hipLaunchKernelGGL(restore_chain_k, dim3(grid_for((size_t)Mmax, 4, 8192)), dim3(256), 0, s, x,
                       rbuf, ridx, rslot, cur, src, Mdev, F, N, D, G);
}

void launch_copy_ref_kv(const void* qkv, const int* pos, int f, int N, int D, int el, void* dst,
                        hipStream_t s) {
    hipLaunchKernelGGL(copy_ref_kv_k, dim3(grid_for((size_t)N * 2 * D * el / 16, 256)), dim3(256),
                       0, s, qkv, pos, f, N, D, el, dst);
}

void launch_copy_rows(const float* x, const int* root, int f, int N, int D, float* dst,
                      hipStream_t s) {
    hipLaunchKernelGGL(copy_rows_k, dim3(grid_for((size_t)N, 4)), dim3(256), 0, s, x, root, f, N,
                       D, dst);
}

void launch_ln_rows(bool bf16, const float* src, const int* gather, const int* Mdev, int Mmax,
                    int D, const float* g, const float* b, void* dst, hipStream_t s) {
    const int grid = grid_for((size_t)Mmax, 4, 65536);
    // rows of at most 1024 values: 4 float4 chunks per lane in registers, else up to 8
    auto k = bf16 ? (D <= 1024 ? ln_rows_k<true, 4> : D <= 1280 ? ln_rows_k<true, 5> : ln_rows_k<true, 8>)
                  : (D <= 1024 ? ln_rows_k<false, 4> : D <= 1280 ? ln_rows_k<false, 5> : ln_rows_k<false, 8>);
    hipLaunchKernelGGL(k, dim3(grid), dim3(256), 0, s, src, gather, Mdev, Mmax, D, g, b, dst);
}

void launch_merge(float* x, const uint8_t* cur, const int* root, int F, int N, int D, int G,
                  hipStream_t s) {
    hipLaunchKernelGGL(merge_k, dim3(grid_for((size_t)F * N, 4, 4096)), dim3(256), 0, s, x, cur,
                       root, F, N, D, G);
}

void launch_resolve(const uint8_t* cur, const uint8_t* src, int F, int N, int G, int* pos,
                    int* root, hipStream_t s) {
    hipLaunchKernelGGL(resolve_k, dim3(grid_for((size_t)F * N, 256)), dim3(256), 0, s, cur, src,
                       F, N, G, pos, root);
}

void launch_final_ln(const float* x, int F, int N, int D, const float* g, const float* b,
                     float* emb, hipStream_t s) {
    hipLaunchKernelGGL(final_ln_k, dim3(grid_for((size_t)F, 4)), dim3(256), 0, s, x, F, N, D, g,
                       b, emb);
}

void launch_fill_u8(uint8_t* p, size_t n, uint8_t v, hipStream_t s) {
    hipLaunchKernelGGL(fill_u8_k, dim3(grid_for(n, 256)), dim3(256), 0, s, p, n, v);
}

void launch_zero_mask_layer(uint8_t* om, int F, int L, int N, int layer, hipStream_t s) {
    hipLaunchKernelGGL(zero_mask_layer_k, dim3(grid_for((size_t)F * N, 256)), dim3(256), 0, s, om,
                       F, L, N, layer);
}

}  // namespace dv
