// Attention over mixed fresh and reference K/V.
//
// Per-frame kernel: one block per (frame f, head h).  The block stages the frame's N keys and
// values of head h in LDS, reading each key row through pos[]: a recomputed token's own packed
// row, or -- for a reused token -- the packed row of the same token of the reference frame.
// The frame's packed query rows qoff[f] .. qoff[f+1] are cut into tiles of 32 that the
// block's wavefronts take in turn.  Per-unit kernel (star groups): the reference's keys are
// staged once for all frames of a group.  Per-tile kernel (reuse without groups: reordering,
// stream calls): a wavefront takes one or two query tiles of a frame and streams the keys
// through its own LDS buffer.
//
// bf16 path (MFMA 32x32x16, fp32 accumulate), every quantity kept with one query per lane:
//   S^T = K . Q^T      A = K rows from LDS, B = the query tile (registers); lane l holds the
//                      scores of query l%32 against 16 of the 32 keys of a key block
//   online softmax     max / sum over a lane's 16 registers plus one shuffle with lane l^32
//   O^T += V^T . P^T   A = V^T, read from row-major V with the transposing LDS read
//                      ds_read_b64_tr_b16; B = the probabilities as they sit in the S^T
//                      accumulators; the contraction runs over the 32 keys in the order the
//                      accumulator layout gives (the same order on both operands)
// so a lane rescales and normalises its own query's output without any shuffle.  A query tile is
// always taken by one wavefront over all key blocks in order, whatever kernel runs it and however
// many other queries its frame has, so a row's result depends only on its query and the frame's
// keys and values (no split of the keys across wavefronts, whose merge would round the
// probabilities against partial maxima).
//
// fp32 path: scalar scores, softmax and P.V (small fp32 models).
#include <algorithm>
#include <cstdlib>
#include <type_traits>

#include "dv_internal.h"

namespace dv {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int NWAVE = 4;

__device__ inline void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Workgroup barrier that orders LDS only: this wave's LDS operations are complete and every
// wave has arrived.  Unlike __syncthreads() it does not wait for global stores in flight, so
// the output rows of one work item drain while the next item is staged.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

__device__ inline float wmax(float v) {
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}
__device__ inline float wsum(float v) {
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// ---- LDS geometry of the bf16 kernel (shared by host sizing and the kernel) ------------------
// K rows: the MFMA reads 16 bytes (one chunk) of 16 consecutive rows; V rows: the transposing
// read ds_read_b64_tr_b16 reads 8 bytes (4 dims) of 4 consecutive keys x 4 dim-words.  Row
// strides and XOR swizzles (in 16-byte chunks) keep both patterns on distinct banks:
//   head dim 64:  K chunk c of row r at c ^ ((r>>1)&7),  V chunk c of row j at c ^ 2((j>>1)&3)
//   head dim 128: K chunk c of row r at c ^ (r&15),      V chunk c of row j at c ^ 2(j&3)
//   head dim 80/96: no swizzle; K rows padded to dh+8, V rows to 96 elements.
struct Geo {
    int npad, dhp, ldk, ldv, dh;
    __host__ __device__ Geo(int N, int d) : dh(d) {
        npad = (N + 31) / 32 * 32;
        dhp = (d + 31) / 32 * 32;
        ldk = (d == 64 || d == 128) ? d : d + 8;
        ldv = (d == 64 || d == 128) ? d : 96;
    }
    __host__ __device__ int kofs(int r, int c) const {
        const int x = dh == 64 ? ((r >> 1) & 7) : dh == 128 ? (r & 15) : 0;
        return r * ldk + (c ^ x) * 8;
    }
    __host__ __device__ int vofs(int j, int c) const {
        const int x = dh == 64 ? 2 * ((j >> 1) & 3) : dh == 128 ? 2 * (j & 3) : 0;
        return j * ldv + (c ^ x) * 8;
    }
    __host__ __device__ size_t bytes() const {
        return ((size_t)npad * ldk + (size_t)npad * ldv) * 2;
    }
};

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

// four floats to four bf16 (round to nearest even, v_cvt_pk_bf16_f32)
__device__ inline uint2 pack_bf16x4(float a, float b, float c, float d) {
    const bf16x4 v = {(__bf16)a, (__bf16)b, (__bf16)c, (__bf16)d};
    return __builtin_bit_cast(uint2, v);
}
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));   // native vector: stays in VGPRs

// The value a lane's partner in the other half of the wavefront (lane l ^ 32) holds.
__device__ inline float other_half(float x) {
    const unsigned u = __builtin_bit_cast(unsigned, x);
    const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    return __builtin_bit_cast(float, (threadIdx.x & 32) ? r[0] : r[1]);
}

constexpr int AW = 8;    // wavefronts of a per-frame attention block
constexpr int UW = 12;   // wavefronts of a per-unit attention block

// Online-softmax attention of one query tile (fragments qf, one query per lane) against the
// staged K/V: key blocks taken two at a time in order (kb, kb + 1) -- two independent MFMA
// chains and at most one rescale per step.  krow maps a key to its LDS row; stage(kb) runs
// before the step of blocks kb, kb + 1 reads them (a kernel streaming K/V through LDS loads them
// there).  On return (m, l, o) hold the maximum the tile's probabilities are scaled to (raw score
// units; at most 8 / sl2 below the running maximum), their sum and the unnormalised output.  The
// arithmetic and its order depend only on the key values, never on where the rows sit.
template <int DH, class KRow, class Stage>
__device__ __forceinline__ void attend_tile(const Geo& g, const uint16_t* Ks, const uint16_t* Vs,
                                            int N, int lane, const bf16x8 (&qf)[DH / 16],
                                            KRow krow, float& m, float& l,
                                            f32x16 (&o)[(DH + 31) / 32], Stage stage) {
    constexpr int KS = DH / 16;          // k-steps of S^T
    constexpr int DB = (DH + 31) / 32;   // 32-row blocks of O^T
    const int hl = lane >> 5, lr = lane & 31;
    const float sl2 = 1.4426950408889634f / sqrtf((float)DH);  // log2(e) / sqrt(dh)
    const float lazy = 8.0f / sl2;    // raw score units of a factor 2^8
    const int nkb = g.npad / 32;
    const int grp = lane >> 4, gi = lane & 15;    // 16-lane group of the transposing read
    const int tr_key = hl * 4 + (gi >> 2);
    const int tr_dim = (grp & 1) * 16 + (gi & 3) * 4;

    // scores of key block kb against the query tile (raw, unscaled); MK: the block may hold
    // keys past N
    auto scores = [&](int kb, auto mk) {
        f32x16 sc;
#pragma unroll
        for (int r = 0; r < 16; ++r) sc[r] = 0.f;
        const int row = krow(kb * 32 + lr);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const bf16x8 kf = *(const bf16x8*)(Ks + g.kofs(row, ks * 2 + hl));
            sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], sc, 0, 0, 0);
        }
        if (decltype(mk)::value && (kb + 1) * 32 > N) {   // ragged last block: keys past N get -inf
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int key = kb * 32 + (r >> 2) * 8 + hl * 4 + (r & 3);
                sc[r] = key < N ? sc[r] : -INFINITY;
            }
        }
        return sc;
    };
    // O^T += V^T(kb) . P^T(kb)
    auto accumulate = [&](int kb, const bf16x8 (&pf)[2]) {
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            // lane (group grp, index gi) names key kb*32 + ks*16 + hl*4 + gi/4 (+8) and dims
            // b*32 + (grp&1)*16 + 4*(gi%4); it receives dim b*32 + (grp&1)*16 + gi of the 4
            // keys named by lanes 4e + gi/4 of its group
            const int key = kb * 32 + ks * 16 + tr_key;
            const int r0 = krow(key), r1 = krow(key + 8);
#pragma unroll
            for (int b = 0; b < DB; ++b) {
                int d = b * 32 + tr_dim;
                d = d < DH ? d : DH - 4;   // head dims past DH: any finite row data
                const uint16_t* p0 = Vs + g.vofs(r0, d >> 3) + (d & 7);
                const uint16_t* p1 = Vs + g.vofs(r1, d >> 3) + (d & 7);
                const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) s16x4*)p0);
                const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) s16x4*)p1);
                const s16x4 both[2] = {lo, hi};
                const bf16x8 vf = __builtin_bit_cast(bf16x8, both);
                o[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[ks], o[b], 0, 0, 0);
            }
        }
    };

#pragma unroll
    for (int b = 0; b < DB; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[b][r] = 0.f;
    m = -INFINITY;
    l = 0.f;
    // One softmax step over key blocks kb and kb + 1.  MK: the step may hold the ragged last
    // block or no second block; only the loop's tail steps do, so the others carry no per-key
    // test (the arithmetic and its order are the same either way).
    auto step = [&](int kb, auto mk) {
        constexpr bool MK = decltype(mk)::value;
        stage(kb);
        const int kb1 = kb + 1;
        const bool two = !MK || kb1 < nkb;
        const f32x16 s0 = scores(kb, mk);
        f32x16 s1;
        if (two) {
            s1 = scores(kb1, mk);
        } else {
#pragma unroll
            for (int r = 0; r < 16; ++r) s1[r] = -INFINITY;
        }
        // block maximum and, below, the probability sum as pairwise trees (short dependency
        // chains; the maximum is exact in any order)
        float mx[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) mx[r] = fmaxf(s0[r], s1[r]);
#pragma unroll
        for (int w = 8; w >= 1; w >>= 1)
#pragma unroll
            for (int r = 0; r < w; ++r) mx[r] = fmaxf(mx[r], mx[r + w]);
        float bm = mx[0];
        bm = fmaxf(bm, other_half(bm));
        // rescale only when some lane's block maximum passes its reference maximum m by more
        // than 8 in log2 units: probabilities stay below 2^8 (far inside the range of the fp32
        // sums and bf16 products), and most steps after the first keep their scale
        if (__any(bm > m + lazy)) {
            const float mn = fmaxf(m, bm);
            const float alpha = __builtin_amdgcn_exp2f((m - mn) * sl2);
            l *= alpha;
#pragma unroll
            for (int b = 0; b < DB; ++b)
#pragma unroll
                for (int r = 0; r < 16; ++r) o[b][r] *= alpha;
            m = mn;
        }
        const float nm = -m * sl2;
        float sr[16];
        bf16x8 p0[2], p1[2];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const float e0 = __builtin_amdgcn_exp2f(fmaf(s0[r], sl2, nm));
            const float e1 = __builtin_amdgcn_exp2f(fmaf(s1[r], sl2, nm));
            sr[r] = e0 + e1;
            p0[r >> 3][r & 7] = (__bf16)e0;
            p1[r >> 3][r & 7] = (__bf16)e1;
        }
#pragma unroll
        for (int w = 8; w >= 1; w >>= 1)
#pragma unroll
            for (int r = 0; r < w; ++r) sr[r] += sr[r + w];
        const float ps = sr[0];
        l += ps + other_half(ps);
        accumulate(kb, p0);
        if (two) accumulate(kb1, p1);
    };
    const int nfull = N / 32;   // key blocks with no key past N
    int kb = 0;
    for (; kb + 1 < nfull; kb += 2) step(kb, std::integral_constant<bool, false>());
    for (; kb < nkb; kb += 2) step(kb, std::integral_constant<bool, true>());
}

// attend_tile for up to NQ query tiles of one frame at once (nq of them present): every step's
// keys and values are staged once for all of them; each tile's arithmetic, in its order, is
// attend_tile's, so its results are the same bit for bit.
template <int DH, int NQ, class KRow, class Stage>
__device__ __forceinline__ void attend_tiles(const Geo& g, const uint16_t* Ks, const uint16_t* Vs,
                                             int N, int lane, const bf16x8 (&qf)[NQ][DH / 16],
                                             int nq, KRow krow, float (&m)[NQ], float (&l)[NQ],
                                             f32x16 (&o)[NQ][(DH + 31) / 32], Stage stage) {
    constexpr int KS = DH / 16;          // k-steps of S^T
    constexpr int DB = (DH + 31) / 32;   // 32-row blocks of O^T
    const int hl = lane >> 5, lr = lane & 31;
    const float sl2 = 1.4426950408889634f / sqrtf((float)DH);  // log2(e) / sqrt(dh)
    const float lazy = 8.0f / sl2;    // raw score units of a factor 2^8
    const int nkb = g.npad / 32;
    const int grp = lane >> 4, gi = lane & 15;    // 16-lane group of the transposing read
    const int tr_key = hl * 4 + (gi >> 2);
    const int tr_dim = (grp & 1) * 16 + (gi & 3) * 4;

    // scores of key block kb against the query tile (raw, unscaled); MK: the block may hold
    // keys past N
    auto scores = [&](int q, int kb, auto mk) {
        f32x16 sc;
#pragma unroll
        for (int r = 0; r < 16; ++r) sc[r] = 0.f;
        const int row = krow(kb * 32 + lr);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const bf16x8 kf = *(const bf16x8*)(Ks + g.kofs(row, ks * 2 + hl));
            sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[q][ks], sc, 0, 0, 0);
        }
        if (decltype(mk)::value && (kb + 1) * 32 > N) {   // ragged last block: keys past N get -inf
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int key = kb * 32 + (r >> 2) * 8 + hl * 4 + (r & 3);
                sc[r] = key < N ? sc[r] : -INFINITY;
            }
        }
        return sc;
    };
    // O^T += V^T(kb) . P^T(kb)
    auto accumulate = [&](int q, int kb, const bf16x8 (&pf)[2]) {
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            // lane (group grp, index gi) names key kb*32 + ks*16 + hl*4 + gi/4 (+8) and dims
            // b*32 + (grp&1)*16 + 4*(gi%4); it receives dim b*32 + (grp&1)*16 + gi of the 4
            // keys named by lanes 4e + gi/4 of its group
            const int key = kb * 32 + ks * 16 + tr_key;
            const int r0 = krow(key), r1 = krow(key + 8);
#pragma unroll
            for (int b = 0; b < DB; ++b) {
                int d = b * 32 + tr_dim;
                d = d < DH ? d : DH - 4;   // head dims past DH: any finite row data
                const uint16_t* p0 = Vs + g.vofs(r0, d >> 3) + (d & 7);
                const uint16_t* p1 = Vs + g.vofs(r1, d >> 3) + (d & 7);
                const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) s16x4*)p0);
                const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) s16x4*)p1);
                const s16x4 both[2] = {lo, hi};
                const bf16x8 vf = __builtin_bit_cast(bf16x8, both);
                o[q][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[ks], o[q][b], 0, 0, 0);
            }
        }
    };

#pragma unroll
    for (int q = 0; q < NQ; ++q) {
#pragma unroll
        for (int b = 0; b < DB; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) o[q][b][r] = 0.f;
        m[q] = -INFINITY;
        l[q] = 0.f;
    }
    // one step over key blocks kb, kb + 1 for every tile; MK as in attend_tile
    auto step = [&](int kb, auto mk) {
        constexpr bool MK = decltype(mk)::value;
        stage(kb);
        const int kb1 = kb + 1;
        const bool two = !MK || kb1 < nkb;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            if (q >= nq) break;   // wave-uniform: the tile does not exist
            const f32x16 s0 = scores(q, kb, mk);
            f32x16 s1;
            if (two) {
                s1 = scores(q, kb1, mk);
            } else {
#pragma unroll
                for (int r = 0; r < 16; ++r) s1[r] = -INFINITY;
            }
            float mx[16];   // as in attend_tile: pairwise trees
#pragma unroll
            for (int r = 0; r < 16; ++r) mx[r] = fmaxf(s0[r], s1[r]);
#pragma unroll
            for (int w = 8; w >= 1; w >>= 1)
#pragma unroll
                for (int r = 0; r < w; ++r) mx[r] = fmaxf(mx[r], mx[r + w]);
            float bm = mx[0];
            bm = fmaxf(bm, other_half(bm));
            if (__any(bm > m[q] + lazy)) {   // as in attend_tile
                const float mn = fmaxf(m[q], bm);
                const float alpha = __builtin_amdgcn_exp2f((m[q] - mn) * sl2);
                l[q] *= alpha;
#pragma unroll
                for (int b = 0; b < DB; ++b)
#pragma unroll
                    for (int r = 0; r < 16; ++r) o[q][b][r] *= alpha;
                m[q] = mn;
            }
            const float nm = -m[q] * sl2;
            float sr[16];
            bf16x8 p0[2], p1[2];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float e0 = __builtin_amdgcn_exp2f(fmaf(s0[r], sl2, nm));
                const float e1 = __builtin_amdgcn_exp2f(fmaf(s1[r], sl2, nm));
                sr[r] = e0 + e1;
                p0[r >> 3][r & 7] = (__bf16)e0;
                p1[r >> 3][r & 7] = (__bf16)e1;
            }
#pragma unroll
            for (int w = 8; w >= 1; w >>= 1)
#pragma unroll
                for (int r = 0; r < w; ++r) sr[r] += sr[r + w];
            const float ps = sr[0];
            l[q] += ps + other_half(ps);
            accumulate(q, kb, p0);
            if (two) accumulate(q, kb1, p1);
        }
    };
    const int nfull = N / 32;   // key blocks with no key past N
    int kb = 0;
    for (; kb + 1 < nfull; kb += 2) step(kb, std::integral_constant<bool, false>());
    for (; kb < nkb; kb += 2) step(kb, std::integral_constant<bool, true>());
}

// o / l of a lane's query as bf16 to its output row (dims of this lane's register groups)
template <int DH>
__device__ __forceinline__ void store_row(uint16_t* dst, int lane, float l,
                                          const f32x16 (&o)[(DH + 31) / 32]) {
    constexpr int DB = (DH + 31) / 32;
    const int hl = lane >> 5;
    const float inv = 1.0f / l;
#pragma unroll
    for (int b = 0; b < DB; ++b)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
            const int d = b * 32 + q4 * 8 + hl * 4;
            if (d < DH)
                *(uint2*)(dst + d) = pack_bf16x4(o[b][q4 * 4 + 0] * inv, o[b][q4 * 4 + 1] * inv,
                                                 o[b][q4 * 4 + 2] * inv, o[b][q4 * 4 + 3] * inv);
        }
}

// ---- per-frame items ---------------------------------------------------------------------------
// Work split: T = ceil(q/32) query tiles over AW wavefronts, each tile over all key blocks.
template <int DH>
__device__ __forceinline__ void attn_item(const AttnArgs& a, int f, int h, char* smem);

template <int DH>
__global__ __launch_bounds__(AW * 64) __attribute__((amdgpu_waves_per_eu(DH == 64 ? 4 : 2, DH == 64 ? 4 : 2)))
void attn_mfma_k(AttnArgs a) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    // The grid holds as many blocks as are resident at once (a multiple of 8, one share per
    // XCD) and each block walks a list of work items (frame f, head h): one item per launch slot
    // would leave the compute units waiting on workgroup dispatch when items are short.
    // Without groups the items are striped over the blocks, heads fastest, so that the items of a
    // frame land on all 8 XCDs (block i runs on XCD i % 8; with frames fastest, every I frame of
    // a reordered batch, one frame in 8, would fall on the same XCD).  With groups, a unit
    // (a group's frames, one head) lives on XCD unit % 8, whose L2 then serves the reference
    // rows all of its frames read; the units of XCD x are dealt to its R blocks
    // frame-index-major (entry e = unit e % U, frame e / U of the group), so that every block
    // takes reference and non-reference frames alike.
    if (a.G > 0) {
        const int units = (a.F + a.G - 1) / a.G * a.H;
        const int x = blockIdx.x % 8, R = gridDim.x / 8, r = blockIdx.x / 8;
        const int U = (units + 7) / 8;
        for (int e = r; e < U * a.G; e += R) {
            const int u = x + 8 * (e % U), j = e / U;
            const int f = u / a.H * a.G + j;
            if (u < units && f < a.F) attn_item<DH>(a, f, u % a.H, smem);
            lds_barrier();   // the next item restages K/V over this item's LDS
        }
    } else {
        for (int item = blockIdx.x; item < a.F * a.H; item += gridDim.x) {
            attn_item<DH>(a, item / a.H, item % a.H, smem);
            lds_barrier();
        }
    }
}

// One work item: frame f, head h.  Every thread of the block takes the same path.
template <int DH>
__device__ __forceinline__ void attn_item(const AttnArgs& a, int f, int h, char* smem) {
    constexpr int KS = DH / 16;          // k-steps of S^T
    constexpr int DB = (DH + 31) / 32;   // 32-row blocks of O^T
    constexpr int CH = DH / 8;           // 16-byte chunks per row
    constexpr int NT = AW * 64;
    const int N = a.N, D = a.D;
    const Geo g(N, DH);
    uint16_t* Ks = (uint16_t*)smem;
    uint16_t* Vs = Ks + (size_t)g.npad * g.ldk;
    // the thread index passes through an empty asm so that nothing derived from it is hoisted
    // out of the caller's item loop (that would keep it live, and spilled, across items)
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63, wave = tid >> 6;
    const int hl = lane >> 5, lr = lane & 31;
    const size_t ld3 = 3 * (size_t)D;
    const uint16_t* qkv = (const uint16_t*)a.qkv;
    const int q0 = a.qoff[f], q1 = a.qoff[f + 1];
    const int ntile = (q1 - q0 + 31) / 32;
    if (ntile <= a.tile_cut) return;   // none, or taken by per-tile wavefronts

    // stage K and V rows (row-major, 16-byte chunks); keys past N repeat key N-1 (finite data
    // whose scores are masked).  Up to four chunks per thread are gathered before any store.
    const int total = g.npad * CH;
    for (int c0 = tid; c0 < total; c0 += 4 * NT) {
        size_t rowoff[4];
        u32x4 kv[4], vv[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int c = min(c0 + u * NT, total - 1);
            const int j = min(c / CH, N - 1);
            rowoff[u] = (size_t)a.pos[(size_t)f * N + j] * ld3 + h * DH + (c % CH) * 8;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            kv[u] = *(const u32x4*)(qkv + rowoff[u] + D);
            vv[u] = *(const u32x4*)(qkv + rowoff[u] + 2 * D);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int c = c0 + u * NT;
            if (c < total) {
                const int j = c / CH, part = c % CH;
                *(u32x4*)(Ks + g.kofs(j, part)) = kv[u];
                *(u32x4*)(Vs + g.vofs(j, part)) = vv[u];
            }
        }
    }
    lds_barrier();

    float m, l;   // the probabilities' scale (raw score units) and their sum
    f32x16 o[DB];
    for (int t = wave; t < ntile; t += AW) {
        const int myq = q0 + t * 32 + lr;
        const int qrow = myq < q1 ? myq : q1 - 1;   // tail lanes compute on a valid row
        bf16x8 qf[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            qf[ks] = *(const bf16x8*)(qkv + (size_t)qrow * ld3 + h * DH + ks * 16 + hl * 8);
        attend_tile<DH>(g, Ks, Vs, N, lane, qf, [](int k) { return k; }, m, l, o, [](int) {});
        if (myq < q1) store_row<DH>((uint16_t*)a.out + (size_t)myq * D + h * DH, lane, l, o);
    }
}

// ---- per-wavefront items (reuse on: frames with few query tiles) ------------------------------
// A work item is one query tile (frame f, head h, tile t), taken by one wavefront on its own:
// the frame's keys and values stream through a wavefront-private LDS buffer, 64 keys (one step
// of attend_tile) at a time, fetched by buffer_load ... lds through pos (one instruction writes
// 1 KiB: lane i at 16 i, so each lane fetches the chunk that belongs at its slot of the
// swizzled layout).  Nothing is shared between wavefronts -- no barrier -- so a compute unit
// keeps as many tiles in flight as buffers fit, where a per-frame block stages a whole frame
// for what is mostly a single tile.  The arithmetic is attend_tile's: results equal the other
// kernels' bit for bit.
constexpr int SW = 4;   // wavefronts of a per-wavefront attention block

template <int DH>
struct WaveBuf {   // 64 rows of K and 64 of V, with Geo's strides
    static constexpr int LDK = (DH == 64 || DH == 128) ? DH : DH + 8;
    static constexpr int LDV = (DH == 64 || DH == 128) ? DH : 96;
    static constexpr size_t ELEMS = (size_t)64 * (LDK + LDV);
};

template <int DH, int NQ>
__global__ __launch_bounds__(SW * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_wave_k(AttnArgs a) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    constexpr int KS = DH / 16;
    constexpr int DB = (DH + 31) / 32;
    const int N = a.N, D = a.D;
    const Geo g(N, DH);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int hl = lane >> 5, lr = lane & 31;
    using WB = WaveBuf<DH>;
    uint16_t* Ks = (uint16_t*)smem + (size_t)wave * WB::ELEMS;
    uint16_t* Vs = Ks + (size_t)64 * WB::LDK;
    const size_t ld3 = 3 * (size_t)D;
    const uint16_t* qkv = (const uint16_t*)a.qkv;
    // the packed K/V rows (and the cached reference's rows past them) are below 2^32 bytes
    const __amdgpu_buffer_rsrc_t rq =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.qkv), (short)0, (int)0xFFFFFFF0u,
                                          0x00020000);
    static_assert(DH == 64, "rows of 8 16-byte slots, K and V alike");
    constexpr int KI = 8;   // copy instructions per step for K, and as many for V
    // an item is NQ consecutive query tiles of a frame, t .. t + nq - 1
    const int tmax = ((N + 31) / 32 + NQ - 1) / NQ;
    const int items = a.F * a.H * tmax;
    for (int item = blockIdx.x * SW + wave; item < items; item += gridDim.x * SW) {
        const int t = item % tmax * NQ, fh = item / tmax;
        const int f = fh / a.H, h = fh % a.H;
        const int q0 = a.qoff[f], q1 = a.qoff[f + 1];
        if (t * 32 >= q1 - q0 || q1 - q0 > a.tile_cut * 32) continue;   // none, or a per-frame block
        const int nq = min(NQ, (q1 - q0 + 31) / 32 - t);
        const int* pf = a.pos + (size_t)f * N;
        const uint32_t hoff = (uint32_t)(h * DH) * 2;
        // Lane l fetches row r = u*8 + l/8 of instruction u, slot l%8 (K and V rows have the same
        // 8 slots); prow holds those rows' byte offsets for the coming step, loaded one step
        // ahead so that a step waits for one memory round trip (the copy), not two.
        uint32_t prow[KI];
        auto rows = [&](int kb, uint32_t (&dst)[KI]) {
#pragma unroll
            for (int u = 0; u < KI; ++u)
                dst[u] = (uint32_t)pf[min(kb * 32 + u * 8 + (lane >> 3), N - 1)] *
                             (uint32_t)(ld3 * 2) + hoff;
        };
        rows(0, prow);
        // keys kb*32 .. kb*32 + 63 (past N: key N-1, finite data whose scores are masked) into
        // the buffer; LDS row = key - kb*32, the low bits of the key as attend_tile's krow needs
        auto stage = [&](int kb) {
            uint32_t next[KI];
            rows(kb + 2, next);
            __builtin_amdgcn_s_waitcnt(0xc07f);   // this wave's reads of the last step are done
            asm volatile("" ::: "memory");
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                const int r = u * 8 + (lane >> 3), sl = lane & 7;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rq, (__attribute__((address_space(3))) void*)(Ks + u * 512), 16,
                    (int)(prow[u] + (uint32_t)D * 2 + (sl ^ ((r >> 1) & 7)) * 16), 0, 0, 0);
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rq, (__attribute__((address_space(3))) void*)(Vs + u * 512), 16,
                    (int)(prow[u] + (uint32_t)D * 4 + (sl ^ (2 * ((r >> 1) & 3))) * 16), 0, 0,
                    0);
            }
            __builtin_amdgcn_s_waitcnt(0x0070);   // vmcnt(0) lgkmcnt(0): the step has landed
            asm volatile("" ::: "memory");
#pragma unroll
            for (int u = 0; u < KI; ++u) prow[u] = next[u];
        };
        bf16x8 qf[NQ][KS];
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int myq = q0 + (t + q) * 32 + lr;
            const int qrow = myq < q1 ? myq : q1 - 1;   // tail lanes compute on a valid row
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                qf[q][ks] = *(const bf16x8*)(qkv + (size_t)qrow * ld3 + h * DH + ks * 16 + hl * 8);
        }
        float m[NQ], l[NQ];
        f32x16 o[NQ][DB];
        attend_tiles<DH, NQ>(g, Ks, Vs, N, lane, qf, nq, [](int k) { return k & 63; }, m, l, o,
                             stage);
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int myq = q0 + (t + q) * 32 + lr;
            if (q < nq && myq < q1)
                store_row<DH>((uint16_t*)a.out + (size_t)myq * D + h * DH, lane, l[q], o[q]);
        }
    }
}

// ---- per-unit items ----------------------------------------------------------------------------
// A unit is one group of frames and one head.  The reference frame's keys are staged once; a
// non-reference frame reads each reused key from the reference's row and each recomputed key
// from its own row, through a per-frame key -> row map.  A frame's own rows, and those of
// consecutive frames, are consecutive packed rows (stable frame-major compaction; the reference
// frame is recomputed in full, its token i at packed row qoff[f0] + i), so staging is a copy of
// contiguous rows.  Every query tile of the unit goes to one wavefront, over all key blocks:
// no key split and no merge.
//
// LDS: K and V arrays of npad reference rows (keys past N repeat key N-1) followed by up to pcap
// rows of other frames; then one 16-bit key -> row map of npad entries per frame of the group.
struct UnitGeo {
    Geo g;
    int pcap, G;
    __host__ __device__ UnitGeo(int N, int dh, int G_, int pcap_) : g(N, dh), pcap(pcap_), G(G_) {}
    __host__ __device__ int rows() const { return g.npad + pcap; }
    __host__ __device__ size_t vbase() const { return (size_t)rows() * g.ldk; }   // elements
    __host__ __device__ size_t mbase() const { return vbase() + (size_t)rows() * g.ldv; }
    __host__ __device__ size_t bytes() const { return (mbase() + (size_t)G * g.npad) * 2; }
};

// Rows of other frames that fit in `limit` bytes of LDS next to the reference rows and maps.
inline int unit_pcap(int N, int dh, int G, size_t limit) {
    const UnitGeo u(N, dh, G, 0);
    const size_t per = (size_t)(u.g.ldk + u.g.ldv) * 2;
    return u.bytes() >= limit ? 0 : (int)std::min<size_t>((limit - u.bytes()) / per, 32767);
}

// LDS rows dst0 .. dst0+count-1 of K and V <- packed rows src0 + min(i, nvalid - 1), head h
template <int DH, int NT>
__device__ __forceinline__ void stage_rows(const Geo& g, uint16_t* Ks, uint16_t* Vs,
                                           const uint16_t* qkv, size_t ld3, int D, int h, int dst0,
                                           int src0, int count, int nvalid, int tid) {
    constexpr int CH = DH / 8;
    const int total = count * CH;
    for (int c0 = tid; c0 < total; c0 += 4 * NT) {
        u32x4 kv[4], vv[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int c = min(c0 + u * NT, total - 1);
            const size_t off = (size_t)(src0 + min(c / CH, nvalid - 1)) * ld3 + h * DH + (c % CH) * 8;
            kv[u] = *(const u32x4*)(qkv + off + D);
            vv[u] = *(const u32x4*)(qkv + off + 2 * D);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int c = c0 + u * NT;
            if (c < total) {
                const int i = dst0 + c / CH, part = c % CH;
                *(u32x4*)(Ks + g.kofs(i, part)) = kv[u];
                *(u32x4*)(Vs + g.vofs(i, part)) = vv[u];
            }
        }
    }
}

template <int DH>
__global__ __launch_bounds__(UW * 64) __attribute__((amdgpu_waves_per_eu(3, 3)))
void attn_unit_k(AttnArgs a, int pcap) {
    constexpr int KS = DH / 16;
    constexpr int DB = (DH + 31) / 32;
    constexpr int NT = UW * 64;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int G = a.G, N = a.N, D = a.D, H = a.H;
    const UnitGeo ug(N, DH, G, pcap);
    const Geo& g = ug.g;
    uint16_t* Ks = (uint16_t*)smem;
    uint16_t* Vs = Ks + ug.vbase();
    uint16_t* kmap = Ks + ug.mbase();
    const uint16_t* qkv = (const uint16_t*)a.qkv;
    const size_t ld3 = 3 * (size_t)D;
    const int units = (a.F + G - 1) / G * H;
    const int Tref = (N + 31) / 32;   // query tiles of a reference frame
    for (int u = blockIdx.x; u < units; u += gridDim.x) {
        int tid = threadIdx.x;
        asm volatile("" : "+v"(tid));   // keep lane-derived values inside the unit loop
        const int lane = tid & 63, wave = tid >> 6, hl = lane >> 5, lr = lane & 31;
        const int h = u % H, f0 = u / H * G, Gu = min(G, a.F - f0);
        const int r0 = a.qoff[f0];   // the reference frame's token i sits at packed row r0 + i
        stage_rows<DH, NT>(g, Ks, Vs, qkv, ld3, D, h, 0, r0, g.npad, N, tid);
        int Tr = Tref;               // reference tiles not taken yet
        int j = 1;
        do {
            // batch: frames j .. j2-1 of the group whose own rows fit in pcap (every frame's do:
            // pcap >= N), staged after the reference rows
            const int p0 = a.qoff[f0 + j];
            int j2 = j;
            while (j2 < Gu && a.qoff[f0 + j2 + 1] - p0 <= pcap) ++j2;
            const int prow = a.qoff[f0 + j2] - p0;
            if (prow > 0) stage_rows<DH, NT>(g, Ks, Vs, qkv, ld3, D, h, g.npad, p0, prow, prow, tid);
            for (int e = tid; e < (j2 - j) * g.npad; e += NT) {
                const int jj = j + e / g.npad, i = e % g.npad;
                const int p = a.pos[(size_t)(f0 + jj) * N + min(i, N - 1)];
                kmap[jj * g.npad + i] = (uint16_t)(p < r0 + N ? p - r0 : g.npad + p - p0);
            }
            lds_barrier();
            // the batch's tiles, then reference tiles: as many as fill the last round of
            // wavefronts, or all that are left after the last batch
            int Tb = 0;
            for (int jj = j; jj < j2; ++jj) Tb += (a.qoff[f0 + jj + 1] - a.qoff[f0 + jj] + 31) / 32;
            const int extra = j2 >= Gu ? Tr : min(Tr, (UW - Tb % UW) % UW);
            for (int t = wave; t < Tb + extra; t += UW) {
                int jj = -1, tt = t;   // frame (index in the group; -1: the reference) and tile
                if (t < Tb) {
                    jj = j;
                    for (int nt; tt >= (nt = (a.qoff[f0 + jj + 1] - a.qoff[f0 + jj] + 31) / 32); ++jj)
                        tt -= nt;
                } else {
                    tt = Tref - Tr + (t - Tb);
                }
                const int f = jj < 0 ? f0 : f0 + jj;
                const int q0 = a.qoff[f], q1 = a.qoff[f + 1];
                const int myq = q0 + tt * 32 + lr;
                const int qrow = myq < q1 ? myq : q1 - 1;
                bf16x8 qf[KS];
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
                    qf[ks] = *(const bf16x8*)(qkv + (size_t)qrow * ld3 + h * DH + ks * 16 + hl * 8);
                float m, l;
                f32x16 o[DB];
                if (jj < 0) {
                    attend_tile<DH>(g, Ks, Vs, N, lane, qf, [](int k) { return k; }, m, l, o,
                                    [](int) {});
                } else {
                    const uint16_t* km = kmap + jj * g.npad;
                    attend_tile<DH>(g, Ks, Vs, N, lane, qf, [=](int k) { return (int)km[k]; },
                                    m, l, o, [](int) {});
                }
                if (myq < q1) store_row<DH>((uint16_t*)a.out + (size_t)myq * D + h * DH, lane, l, o);
            }
            Tr -= extra;
            lds_barrier();   // the next batch (or unit) restages rows and maps
            j = j2;
        } while (j < Gu);
    }
}

// ---- fp32 path ---------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void attn_f32_k(AttnArgs a) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int f = blockIdx.x, h = blockIdx.y;
    const int N = a.N, D = a.D, dh = D / a.H;
    const int ldk = dh + 1;
    float* Ks = (float*)smem;
    float* Vs = Ks + (size_t)N * ldk;
    float* qs = Vs + (size_t)N * dh;
    float* ps = qs + NWAVE * dh;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const size_t ld3 = 3 * (size_t)D;
    const float* qkv = (const float*)a.qkv;
    for (int e = tid; e < N * dh; e += 256) {
        const int j = e / dh, d = e % dh;
        const size_t row = (size_t)a.pos[(size_t)f * N + j];
        Ks[j * ldk + d] = qkv[row * ld3 + D + h * dh + d];
        Vs[j * dh + d] = qkv[row * ld3 + 2 * D + h * dh + d];
    }
    __syncthreads();
    const float scale = 1.0f / sqrtf((float)dh);
    const int q0 = a.qoff[f], q1 = a.qoff[f + 1];
    float* myq = qs + wave * dh;
    float* myp = ps + wave * N;
    for (int q = q0 + wave; q < q1; q += NWAVE) {
        for (int d = lane; d < dh; d += 64) myq[d] = qkv[(size_t)q * ld3 + h * dh + d] * scale;
        wave_lds_sync();
        float mx = -INFINITY;
        for (int j = lane; j < N; j += 64) {
            float s = 0.f;
            for (int d = 0; d < dh; ++d) s = fmaf(myq[d], Ks[j * ldk + d], s);
            myp[j] = s;
            mx = fmaxf(mx, s);
        }
        mx = wmax(mx);
        float sum = 0.f;
        for (int j = lane; j < N; j += 64) {
            const float p = expf(myp[j] - mx);
            myp[j] = p;
            sum += p;
        }
        sum = wsum(sum);
        wave_lds_sync();
        const float inv = 1.0f / sum;
        for (int d = lane; d < dh; d += 64) {
            float o = 0.f;
            for (int j = 0; j < N; ++j) o = fmaf(myp[j], Vs[j * dh + d], o);
            ((float*)a.out)[(size_t)q * D + h * dh + d] = o * inv;
        }
        wave_lds_sync();  // this wave's myq/myp are rewritten by its next query
    }
}

// ---- class-token attention weights (the decision MLP's importance cue) ------------------------
// One wavefront per (non-reference frame, head): the class query's scores against the frame's N
// keys (read through pos), then their softmax.  Eight lanes share a key: each multiplies one or
// more 16-byte chunks of the key row with the matching chunks of the query (held in registers),
// so a wavefront reads eight key rows per step in whole 128-byte segments; the eight partial
// sums meet in three shuffles.  Four heads per block, no block barriers (each wavefront has its
// own LDS slice).
template <bool BF>
__device__ inline float elem_at(const void* p, size_t i) {
    if constexpr (BF) return bf16_to_f32(((const uint16_t*)p)[i]);
    else return ((const float*)p)[i];
}

template <bool BF>
__global__ __launch_bounds__(256) void cls_attn_k(AttnArgs a, float* __restrict__ out) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    constexpr int CE = BF ? 8 : 4;            // elements per 16-byte chunk
    constexpr int U = 128 / CE / 8;           // chunks per lane for a head dim of up to 128
    constexpr int KB = 4;                     // steps of eight keys whose loads are in flight together
    const int f = blockIdx.x;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int h = blockIdx.y * 4 + wave;
    // reference frames are never gated; frames carried over from an earlier call have no rows
    if ((a.G > 0 && f % a.G == 0) || f < a.skip || h >= a.H) return;
    const int N = a.N, D = a.D, dh = D / a.H, nch = dh / CE;
    const int sub = lane & 7, kq = lane >> 3;
    float* sc = (float*)smem + (size_t)wave * N;   // scores, then exponentials
    const size_t ld3 = 3 * (size_t)D;
    const size_t qrow = (size_t)a.qoff[f] * ld3 + (size_t)h * dh;   // the frame's first row
    float q[U][CE];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < CE; ++e) {
            const int c = sub + 8 * u;
            q[u][e] = c < nch ? elem_at<BF>(a.qkv, qrow + (size_t)c * CE + e) : 0.f;
        }
    const float scale = 1.0f / sqrtf((float)dh);
    typedef typename std::conditional<BF, uint4, float4>::type chunk_t;
    // key rows' packed indices of the steps at j0, loaded one iteration ahead so that an
    // iteration waits for one memory round trip (the key rows), not two
    int pr[KB];
    auto rows_at = [&](int j0, int (&dst)[KB]) {
#pragma unroll
        for (int t = 0; t < KB; ++t) {
            const int j = j0 + 8 * t + kq;
            dst[t] = j < N ? a.pos[(size_t)f * N + j] : 0;
        }
    };
    rows_at(0, pr);
    for (int j0 = 0; j0 < N; j0 += 8 * KB) {
        // KB steps of eight keys at once: every row offset, then every chunk, then the sums
        size_t kr[KB];
#pragma unroll
        for (int t = 0; t < KB; ++t) {
            const int j = j0 + 8 * t + kq;
            kr[t] = j < N ? (size_t)pr[t] * ld3 + D + (size_t)h * dh : 0;
        }
        if (j0 + 8 * KB < N) rows_at(j0 + 8 * KB, pr);
        chunk_t kv[KB][U];
#pragma unroll
        for (int t = 0; t < KB; ++t)
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int c = sub + 8 * u, j = j0 + 8 * t + kq;
                if (j < N && c < nch) {
                    kv[t][u] = *(const chunk_t*)((const char*)a.qkv +
                                                 (kr[t] + (size_t)c * CE) * (BF ? 2 : 4));
                } else {
                    kv[t][u] = chunk_t{0, 0, 0, 0};
                }
            }
#pragma unroll
        for (int t = 0; t < KB; ++t) {
            float s = 0.f;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if constexpr (BF) {
                    const uint32_t w[4] = {kv[t][u].x, kv[t][u].y, kv[t][u].z, kv[t][u].w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        s = fmaf(q[u][2 * e], bf16_to_f32((uint16_t)(w[e] & 0xFFFFu)), s);
                        s = fmaf(q[u][2 * e + 1], bf16_to_f32((uint16_t)(w[e] >> 16)), s);
                    }
                } else {
                    s = fmaf(q[u][0], kv[t][u].x, s);
                    s = fmaf(q[u][1], kv[t][u].y, s);
                    s = fmaf(q[u][2], kv[t][u].z, s);
                    s = fmaf(q[u][3], kv[t][u].w, s);
                }
            }
            s += __shfl_xor(s, 1, 64);
            s += __shfl_xor(s, 2, 64);
            s += __shfl_xor(s, 4, 64);
            const int j = j0 + 8 * t + kq;
            if (sub == 0 && j < N) sc[j] = s * scale;
        }
    }
    wave_lds_sync();
    float mx = -INFINITY;
    for (int j = lane; j < N; j += 64) mx = fmaxf(mx, sc[j]);
    mx = wmax(mx);
    float sum = 0.f;
    for (int j = lane; j < N; j += 64) {
        const float e = expf(sc[j] - mx);
        sc[j] = e;
        sum += e;
    }
    const float inv = 1.0f / wsum(sum);
    float* o = out + ((size_t)f * a.H + h) * N;
    for (int j = lane; j < N; j += 64) o[j] = sc[j] * inv;
}

size_t f32_lds_bytes(int N, int dh) {
    return ((size_t)N * (dh + 1) + (size_t)N * dh + (size_t)NWAVE * dh + (size_t)NWAVE * N) * 4;
}

template <int DH, int NQ>
void launch_wave(const AttnArgs& a, hipStream_t s) {
    constexpr size_t lds = (size_t)SW * WaveBuf<DH>::ELEMS * 2;
    static int per_cu = -1;
    if (per_cu < 0) {
        (void)hipFuncSetAttribute((const void*)attn_wave_k<DH, NQ>,
                                  hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        int v = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&v, (const void*)attn_wave_k<DH, NQ>,
                                                         SW * 64, lds) != hipSuccess)
            v = 0;
        per_cu = v;
    }
    const int items = a.F * a.H * (((a.N + 31) / 32 + NQ - 1) / NQ);
    int grid = (items + SW - 1) / SW;
    if (a.cus > 0 && per_cu > 0) grid = std::min(grid, a.cus * per_cu);
    hipLaunchKernelGGL((attn_wave_k<DH, NQ>), dim3(grid), dim3(SW * 64), lds, s, a);
}

template <int DH>
void launch_bf16(const AttnArgs& a0, hipStream_t s) {
    AttnArgs a = a0;
    a.tile_cut = 0;
    static bool raised = false;
    if (!raised) {  // allow more than the default dynamic LDS (gfx950 has 160 KiB per CU)
        (void)hipFuncSetAttribute((const void*)attn_mfma_k<DH>,
                                  hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        if constexpr (DH == 64)
            (void)hipFuncSetAttribute((const void*)attn_unit_k<DH>,
                                      hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        raised = true;
    }
    // DV_ATTN_CFG (measurements): 1 per-frame blocks only, 2 per-tile wavefronts only, also
    // without reuse, 3 groups too large for per-unit blocks on per-frame blocks placed by unit;
    // DV_ATTN_CUT overrides the cuts below, DV_ATTN_PAIR=0 takes one tile per wavefront.
    static int cfg = -1, cut = -1, pair = 1;
    if (cfg < 0) {
        const char* e = getenv("DV_ATTN_CFG");
        cfg = e ? atoi(e) : 0;
        const char* c = getenv("DV_ATTN_CUT");
        if (c) cut = std::max(0, atoi(c));
        const char* pp = getenv("DV_ATTN_PAIR");
        if (pp) pair = atoi(pp);
    }
    int tcut = cut >= 0 ? cut : 2;
    if constexpr (DH == 64) {
        if (a.G > 1 && a.cus > 0) {
            // groups of several frames: per-unit blocks, one per compute unit, when the
            // reference rows, the maps and at least one other frame's rows fit in LDS
            const int pcap = unit_pcap(a.N, DH, a.G, 160 * 1024);
            if (pcap >= a.N && cfg != 1 && cfg != 2) {
                const size_t lds = UnitGeo(a.N, DH, a.G, pcap).bytes();
                const int units = (a.F + a.G - 1) / a.G * a.H;
                hipLaunchKernelGGL(attn_unit_k<DH>, dim3(std::min(units, a.cus)), dim3(UW * 64),
                                   lds, s, a, pcap);
                return;
            }
            // Otherwise (ViT-L/14 at 336 px: 577 keys) the frames go the way of ungrouped
            // reuse: those with few query tiles to per-tile wavefronts, which read the
            // reference's keys and values through L2 (every frame of a group reads the same
            // rows), the others to per-frame blocks.  Measured at 0 / 34 / 62 / 90 % reuse
            // (attention per 1024-frame encode): per-frame blocks placed by unit 74 / 64 / 56 /
            // 46 ms; cut 2 76 / 63 / 50 / 37; cut 3 78 / 61 / 47 / 35; cut 5 78 / 61 / 51 / 35;
            // every frame per tile 91 / 73 / 51 / 31.  A per-unit kernel over chunks of 64 keys
            // (the reference's chunk rows staged once for the frames of a pass) took 125 / 105 /
            // 89 / 66 ms: its per-chunk barriers serialise staging and the softmax.
            if (cfg != 3) {
                a.G = 0;
                a.sparse = 1;
                tcut = cut >= 0 ? cut : 3;
            }
        }
    }
    // Reuse on without per-group blocks (head dim 64): frames with at most `tcut` query tiles go
    // to per-tile wavefronts streaming K/V (one pass over the keys per tile), the others to
    // per-frame blocks (one staging of the keys for all tiles); of the cuts 2, 3, 4 and 5,
    // 2 gave the shortest attention at 50, 70 and 90 % reuse (ViT-L/14, reordered groups of 8).
    // A wavefront takes two consecutive tiles of a frame at a time, so that a two-tile frame
    // streams its keys once (attention 3.73 / 3.57 / 2.57 ms against 3.75 / 3.67 / 2.70 with
    // one tile per wavefront).
    if constexpr (DH == 64) {
        if (a.G == 0 && cfg != 1 && (a.sparse || cfg == 2)) {
            a.tile_cut = cfg == 2 ? (a.N + 31) / 32 : tcut;
            if (pair) launch_wave<DH, 2>(a, s);
            else launch_wave<DH, 1>(a, s);
            if (a.tile_cut >= (a.N + 31) / 32) return;   // no frame left for per-frame blocks
        }
    }
    const size_t lds = Geo(a.N, DH).bytes();
    // work items: (frame, head) pairs; with reuse, the slots of whole units on each of 8 XCDs
    const int items = a.G > 0 ? xcd_unit_grid((a.F + a.G - 1) / a.G * a.H, a.G) : a.F * a.H;
    static int per_cu = -1;
    if (per_cu < 0) {
        int v = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&v, (const void*)attn_mfma_k<DH>, AW * 64,
                                                         lds) != hipSuccess)
            v = 0;
        per_cu = v;
    }
    // a multiple of 8 blocks keeps item i on XCD i % 8, as the placement of a group's items assumes.
    // After per-tile wavefronts took the small frames, one block per item: the frames left (I
    // frames and others with many recomputed tokens) are spread by the dispatcher, where resident
    // blocks striding over the items would give all of them to a few blocks.
    int grid = items;
    if (a.cus > 0 && per_cu > 0 && a.tile_cut == 0)
        grid = std::min(grid, (a.cus * per_cu + 7) / 8 * 8);
    hipLaunchKernelGGL(attn_mfma_k<DH>, dim3(grid), dim3(AW * 64), lds, s, a);
}

}  // namespace

size_t attention_lds_bytes(bool bf16, int N, int dh) {
    return bf16 ? Geo(N, dh).bytes() : f32_lds_bytes(N, dh);
}

bool attention_supported(bool bf16, int N, int dh) {
    if (attention_lds_bytes(bf16, N, dh) > 160 * 1024) return false;
    if (bf16) return dh == 64 || dh == 80 || dh == 96 || dh == 128;
    return dh % 16 == 0;
}

void launch_cls_attention(bool bf16, const AttnArgs& a, float* probs, hipStream_t s) {
    const size_t lds = 4 * (size_t)a.N * sizeof(float);
    const dim3 grid(a.F, (a.H + 3) / 4);
    if (bf16) hipLaunchKernelGGL(cls_attn_k<true>, grid, dim3(256), lds, s, a, probs);
    else hipLaunchKernelGGL(cls_attn_k<false>, grid, dim3(256), lds, s, a, probs);
}

void launch_attention(bool bf16, const AttnArgs& a, hipStream_t s) {
    const int dh = a.D / a.H;
    if (!bf16) {
        static bool raised = false;
        if (!raised) {
            (void)hipFuncSetAttribute((const void*)attn_f32_k,
                                      hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
            raised = true;
        }
        hipLaunchKernelGGL(attn_f32_k, dim3(a.F, a.H), dim3(256), f32_lds_bytes(a.N, dh), s, a);
        return;
    }
    switch (dh) {
        case 64: launch_bf16<64>(a, s); break;
        case 80: launch_bf16<80>(a, s); break;
        case 96: launch_bf16<96>(a, s); break;
        case 128: launch_bf16<128>(a, s); break;
        default: break;  // rejected at handle creation
    }
}

}  // namespace dv
