// Packed-row GEMMs: C[M, Nout] = A[M, K] * W[Nout, K]^T + fused epilogue.
//
// M (the number of packed recompute rows) lives in device memory; the grid is sized for the
// largest possible M and blocks past the live tiles return at once.
//
// bf16 path: MFMA v_mfma_f32_32x32x16_bf16 with fp32 accumulation.
//   * Block tile BM x BN, 4 wavefronts in 2 x 2, each owning (BM/2) x (BN/2) of 32 x 32 tiles.
//   * k-slices of BK travel global -> LDS with buffer_load_dwordx4 ... lds (no staging registers)
//     through a ring of S stages: S-1 slices are in flight while one is consumed.  One
//     wavefront instruction writes 1 KiB of LDS (lane i at base + 16 i).  LDS rows are BK*2
//     bytes without padding; lane i fetches the global chunk that belongs at its slot: chunk
//     c of tile row r sits at slot c ^ swz(r), so 16 lanes reading one chunk of 16 rows hit
//     distinct banks.
//   * Both operands are K-contiguous rows, so A and B fragments are the same 16-byte LDS read:
//     lane l takes row l%32 and k-slice (l/32)*8 .. +8.  The weight fragment is the MFMA's
//     first operand, so the accumulator is the transposed tile: lane l, register j holds output
//     column (j/4)*8 + (l/32)*4 + j%4 of token row l%32 -- four consecutive columns per
//     register group, stored as one vector by the epilogue.
//   * The fragments of k-step ks+1 are read while the MFMAs of k-step ks run.
//   * Tile order: the live tiles (ceil(M/BM) * Nout/BN) go round-robin over the 8 XCDs in
//     contiguous chunks, each chunk walking groups of 8 tile-rows across all tile-columns, so
//     an XCD's L2 sees few distinct A and W tiles.
//
// fp32 path: a plain LDS-tiled VALU GEMM (small fp32 models).
#include <algorithm>
#include <cstdlib>
#include <type_traits>

#include "dv_internal.h"

namespace dv {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

__device__ inline float gelu_erf(float v) { return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f)); }

// GELU for outputs rounded to bf16: with y = x clamped to [-4, 4], Phi(x) = 1/2 + y P(y^2), P a
// degree-8 least-squares fit to the normal CDF on [0, 4] with 4 P(16) = 1/2 imposed
// (coefficients from gelu_fit.py), so that past |x| = 4 the result is x or 0.  GELU = x Phi(x):
// 12 VALU operations, no transcendental.  |GELU error| <= 1.1e-5 for |x| <= 3 and <= 1.3e-4
// everywhere (largest near |x| = 4): far below the bf16 step (2^-8 relative) of the result.
__device__ inline float gelu_poly(float x) {
    const float y = __builtin_amdgcn_fmed3f(x, -4.0f, 4.0f);
    const float s = y * y;
    float p = 9.151786967e-11f;
    p = fmaf(p, s, -7.699238580e-09f);
    p = fmaf(p, s, 2.898779599e-07f);
    p = fmaf(p, s, -6.548660622e-06f);
    p = fmaf(p, s, 1.009105545e-04f);
    p = fmaf(p, s, -1.142885303e-03f);
    p = fmaf(p, s, 9.898823686e-03f);
    p = fmaf(p, s, -6.643372774e-02f);
    p = fmaf(p, s, 3.989303410e-01f);
    return x * fmaf(y, p, 0.5f);
}

__device__ inline u32x2 pack_bf16x4(f32x4 v) {
    bf16x4 h = {(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};  // v_cvt_pk_bf16_f32 (RNE)
    return __builtin_bit_cast(u32x2, h);
}

template <Epi E, bool BF>
__device__ inline void epi_store(const GemmArgs& a, int row, int col, float acc) {
    float v = acc + a.bias[col];
    if constexpr (E == Epi::Patch) {
        const int f = row / a.P, k = row % a.P;
        const int D = a.Nout;
        v += a.pos[(size_t)(1 + k) * D + col];
        ((float*)a.out)[((size_t)f * a.N + 1 + k) * D + col] = v;
    } else if constexpr (E == Epi::Qkv) {
        if (BF) ((uint16_t*)a.out)[(size_t)row * a.Nout + col] = f32_to_bf16(v);
        else ((float*)a.out)[(size_t)row * a.Nout + col] = v;
    } else if constexpr (E == Epi::OProj) {
        v += a.resid[(size_t)a.idx[row] * a.Nout + col];
        ((float*)a.out)[(size_t)row * a.Nout + col] = v;
    } else if constexpr (E == Epi::Fc1) {
        v = gelu_erf(v);
        if (BF) ((uint16_t*)a.out)[(size_t)row * a.Nout + col] = f32_to_bf16(v);
        else ((float*)a.out)[(size_t)row * a.Nout + col] = v;
    } else if constexpr (E == Epi::Fc2) {
        v += a.resid[(size_t)row * a.Nout + col];
        ((float*)a.out)[(size_t)a.idx[row] * a.Nout + col] = v;
    } else if constexpr (E == Epi::Delta) {
        ((float*)a.out)[(size_t)row * a.Nout + col] = v;
    } else {  // Restore: a reused token's row from its reference token's new row
        const int t = a.idx[row], f = t / a.N;
        const int rt = (f / a.G * a.G) * a.N + t % a.N;
        v += a.resid[(size_t)rt * a.Nout + col];
        ((float*)a.out)[(size_t)t * a.Nout + col] = v;
    }
}

__device__ inline void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Buffer descriptor over `bytes` bytes at p (raw, no stride): a load or store whose 32-bit byte
// offset falls past `bytes` is dropped by the hardware range check.  Every GEMM operand and
// output of the bf16 path is below 2^32 bytes (rows, padding included, are checked at handle
// creation), so offsets are plain 32-bit products and need no 64-bit address arithmetic.
__device__ inline __amdgpu_buffer_rsrc_t buf_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
constexpr uint32_t BUF_ANY = 0xFFFFFFF0u;   // records of a descriptor whose offsets are all valid

// Epilogue of one wavefront's (TI*32) x (TJ*32) sub-tile, staged through a wave-private LDS
// slab so that global traffic is row-contiguous: for each 32-row slab the accumulators (lane l
// holds row l%32, columns (r/4)*8 + (l/32)*4 + r%4 of each 32-column tile) are written to LDS,
// then read back row-major -- each lane owns 4 fixed columns, and a wavefront instruction covers
// 64/(TJ*8) whole row segments.  The accumulators already hold the bias.  Row indices of every
// slab are requested up front and the residual (or position) rows of slab i+1 are in flight
// while slab i is combined and stored.  Stores go through buffer descriptors: rows past M in
// the tile tail get an offset past the descriptor and are dropped.  The caller has finished
// with the LDS ring.
template <Epi E, int TI, int TJ>
__device__ inline void epilogue_lds(const GemmArgs& a, f32x16 (&acc)[TI][TJ], float* slab, int row0,
                                    int col0, int M, int lane) {
    constexpr int WN = TJ * 32;          // columns of the sub-tile
    constexpr int LDW = WN + 4;          // padded slab row (floats)
    constexpr int CPRW = WN / 4;         // 16-byte chunks per row
    constexpr int RPI = 64 / CPRW;       // rows per wavefront instruction
    constexpr int NQ = 32 / RPI;         // instructions per 32-row slab
    constexpr bool LOADS = E == Epi::OProj || E == Epi::Fc2 || E == Epi::Patch || E == Epi::Restore;
    // output rows are token rows
    constexpr bool SCATTER = E == Epi::Fc2 || E == Epi::Patch || E == Epi::Restore;
    constexpr uint32_t ESZ = (E == Epi::Qkv || E == Epi::Fc1) ? 2 : 4;   // output element bytes
    const int lr = lane & 31, hl = lane >> 5;
    const int c = lane % CPRW, rsub = lane / CPRW;
    const uint32_t col = col0 + c * 4;
    const uint32_t Nout = a.Nout;
    // packed-row outputs end at row M; token-row outputs drop tail rows by their offset
    const auto rout = buf_rsrc(a.out, SCATTER ? BUF_ANY : (uint32_t)M * Nout * ESZ);
    const auto rres = buf_rsrc(E == Epi::Patch ? (const void*)a.pos : (const void*)a.resid, BUF_ANY);

    auto row_of = [&](int i, int q) { return row0 + i * 32 + q * RPI + rsub; };
    // residual (or position) rows and output offsets of slab i; one slab ahead
    f32x4 extra[2][NQ];
    uint32_t ooff[2][NQ];
    auto fetch = [&](int i, f32x4 (&dst)[NQ], uint32_t (&oo)[NQ]) {
        int tr[NQ];
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int row = row_of(i, q);
            const int r = row < M ? row : M - 1;           // a valid row for the tile tail
            if constexpr (E == Epi::OProj || E == Epi::Fc2 || E == Epi::Restore) tr[q] = a.idx[r];
            else if constexpr (E == Epi::Patch) tr[q] = (r / a.P) * a.N + 1 + r % a.P;
            else tr[q] = row;
        }
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int row = row_of(i, q);
            if constexpr (SCATTER)
                oo[q] = row < M ? ((uint32_t)tr[q] * Nout + col) * ESZ : BUF_ANY;
            else
                oo[q] = ((uint32_t)row * Nout + col) * ESZ;
        }
        if constexpr (LOADS) {
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                const int row = row_of(i, q);
                const uint32_t r = row < M ? row : M - 1;
                uint32_t off;
                if constexpr (E == Epi::OProj) {
                    off = ((uint32_t)tr[q] * Nout + col) * 4;
                } else if constexpr (E == Epi::Fc2) {
                    off = (r * Nout + col) * 4;
                } else if constexpr (E == Epi::Restore) {   // the reference token's row
                    const uint32_t t = tr[q], f = t / a.N;
                    off = (((f / a.G * a.G) * a.N + t % a.N) * Nout + col) * 4;
                } else {
                    off = ((1 + r % a.P) * Nout + col) * 4;
                }
                dst[q] = __builtin_amdgcn_raw_buffer_load_b128(rres, (int)off, 0, 0);
            }
        }
    };
    fetch(0, extra[0], ooff[0]);
#pragma unroll
    for (int i = 0; i < TI; ++i) {
        if (i + 1 < TI) fetch(i + 1, extra[(i + 1) & 1], ooff[(i + 1) & 1]);
#pragma unroll
        for (int j = 0; j < TJ; ++j)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                f32x4 v = {acc[i][j][g * 4 + 0], acc[i][j][g * 4 + 1], acc[i][j][g * 4 + 2],
                           acc[i][j][g * 4 + 3]};
                *(f32x4*)(slab + lr * LDW + j * 32 + g * 8 + hl * 4) = v;
            }
        wave_lds_sync();
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int r = q * RPI + rsub;
            const f32x4 v = *(const f32x4*)(slab + r * LDW + c * 4);   // bias included
            const int off = (int)ooff[i & 1][q];
            if constexpr (E == Epi::Qkv) {
                __builtin_amdgcn_raw_buffer_store_b64(pack_bf16x4(v), rout, off, 0, 0);
            } else if constexpr (E == Epi::Fc1) {
                const f32x4 gl = {gelu_poly(v[0]), gelu_poly(v[1]), gelu_poly(v[2]), gelu_poly(v[3])};
                __builtin_amdgcn_raw_buffer_store_b64(pack_bf16x4(gl), rout, off, 0, 0);
            } else if constexpr (E == Epi::Delta) {
                __builtin_amdgcn_raw_buffer_store_b128(v, rout, off, 0, 0);
            } else {
                __builtin_amdgcn_raw_buffer_store_b128(v + extra[i & 1][q], rout, off, 0, 0);
            }
        }
        wave_lds_sync();   // the slab is rewritten by the next 32-row slab
    }
}

// s_waitcnt vmcnt(n) lgkmcnt(0) (gfx9 encoding: vmcnt in bits 3:0 and 15:14, expcnt 6:4 left
// at its maximum, lgkmcnt 11:8): all of this wave's loads but the last n have landed in LDS and
// its own LDS reads are complete.
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt(0x0070 | (N & 15) | ((N >> 4) << 14));
}

// Workgroup barrier without the memory fence of __syncthreads() (that fence would wait for
// every load in flight, i.e. drain the LDS ring).  Callers order memory with wait_vm first; the
// signal fences stop the compiler from moving memory accesses across the barrier.
__device__ __forceinline__ void bare_barrier() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Tile of launch index bid among mt x tilesN live tiles: the tiles go round-robin over the 8 XCDs
// in contiguous chunks, each chunk walking groups of 8 tile-rows across all tile-columns, so an
// XCD's L2 sees few distinct A and W tiles at a time.
__device__ __forceinline__ void tile_coords(int bid, int mt, int tilesN, int& tm, int& tn) {
    const int active = mt * tilesN;
    int lid = bid;
    const int per = active / 8;
    if (bid < per * 8) lid = (bid % 8) * per + bid / 8;
    constexpr int GM = 8;
    const int group = lid / (GM * tilesN);
    const int first_m = group * GM;
    const int gsize = min(mt - first_m, GM);
    const int w_in = lid - group * GM * tilesN;
    tm = first_m + w_in % gsize;
    tn = w_in / gsize;
}

// ---------------- bf16 MFMA GEMM, pipelined ----------------------------------------------------
// One block tile of a wave group: the DMA ring keeps S-1 k-slices in flight and the MFMA
// fragments are always one k-step ahead, across stage boundaries too.  The barrier of stage
// kt+1 sits just before the first fragment loads of stage kt+1; the DMA of a new stage is issued
// right after it, into the slot every wave finished reading before that barrier.  The tile is
// number `bid` of the rows [m0, M); `sm` is the group's LDS and `wave` its index in the group.
// Every wavefront of the workgroup passes the same barriers (a group without a tile has left).
// PERSIST: the block goes on to tiles bid + stride, bid + 2 stride, ... of the same rows; when a
// tile's last k-slice starts, the next tile's first slice and bias are copied into the ring slot
// that is then free, and the epilogue's slabs sit past that slot.
template <Epi E, int BM, int BN, int BKD, int S, int WGM, int WGN, bool PERSIST = false>
__device__ __forceinline__ void pipe_tile(const GemmArgs& a, uint16_t* sm, int bid, int m0, int M,
                                          int wave, int stride = 0) {
    constexpr int NW = WGM * WGN;                 // wavefronts, WGM x WGN over the block tile
    constexpr int WM = BM / WGM, WN = BN / WGN, TI = WM / 32, TJ = WN / 32;
    constexpr int CPR = BKD / 8;
    constexpr int RPI = 64 / CPR;
    constexpr int SH = (CPR == 8) ? 1 : 2;
    constexpr int LA = BM / RPI / NW, LB = BN / RPI / NW;
    static_assert(LA * RPI * NW == BM && LB * RPI * NW == BN, "load split");
    constexpr int L = LA + LB;
    constexpr int STAGE = (BM + BN) * BKD;
    constexpr int KS = BKD / 16;
    static_assert(KS % 2 == 0, "fragment double buffer assumes an even number of k-steps");

    const int tilesN = a.Nout / BN;
    const int mt = (M - m0 + BM - 1) / BM;
    const int active = mt * tilesN;
    if (bid >= active) return;
    int tm, tn;

    const int lane = threadIdx.x & 63;
    const int wm = wave / WGN, wn = wave % WGN;
    const int lr = lane & 31, hl = lane >> 5;
    const int K = a.K;

    // this lane's DMA chunks: 32-bit byte offsets into the A and weight buffers (both below 2^32
    // bytes); the k-slice advance rides in the scalar offset of buffer_load ... lds
    const int lrow = lane / CPR, lslot = lane % CPR;
    uint32_t goffA[LA], goffB[LB];
    auto setup = [&](int b, int& tm_, int& tn_) {
        tile_coords(b, mt, tilesN, tm_, tn_);
#pragma unroll
        for (int t = 0; t < LA; ++t) {
            const int r = (wave * LA + t) * RPI + lrow;
            const int c = lslot ^ ((r >> SH) & (CPR - 1));
            const int grow = m0 + tm_ * BM + r;
            const int arow = a.a_idx ? (grow < M ? a.a_idx[grow] : 0) : grow;   // gathered A rows
            goffA[t] = ((uint32_t)arow * K + c * 8) * 2;
        }
#pragma unroll
        for (int t = 0; t < LB; ++t) {
            const int r = (wave * LB + t) * RPI + lrow;
            const int c = lslot ^ ((r >> SH) & (CPR - 1));
            goffB[t] = ((uint32_t)(tn_ * BN + r) * K + c * 8) * 2;
        }
    };
    setup(bid, tm, tn);
    const auto rA = buf_rsrc(a.A, BUF_ANY);
    const auto rW = buf_rsrc(a.W, BUF_ANY);
    const auto rBias = buf_rsrc(a.bias, BUF_ANY);
    auto issue = [&](int kt) {
        uint16_t* st = sm + (kt % S) * STAGE;
        const int soff = kt * BKD * 2;
#pragma unroll
        for (int t = 0; t < LA; ++t)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rA,
                (__attribute__((address_space(3))) void*)(st + (wave * LA + t) * RPI * BKD), 16,
                (int)goffA[t], soff, 0, 0);
#pragma unroll
        for (int t = 0; t < LB; ++t)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rW,
                (__attribute__((address_space(3))) void*)(st + BM * BKD + (wave * LB + t) * RPI * BKD), 16,
                (int)goffB[t], soff, 0, 0);
    };
    // persistent tiles: the tile's bias (BN floats) goes to LDS past the slabs with the DMA of its
    // first slice, so that setting the accumulators waits on no vector memory operation (a
    // global load there would also wait for the previous epilogue's stores)
    constexpr size_t RING_B = (size_t)S * STAGE * 2;
    constexpr size_t SLAB_END = (size_t)STAGE * 2 + (size_t)NW * 32 * (TJ * 32 + 4) * 4;
    float* const bias_lds = (float*)((char*)sm + (RING_B > SLAB_END ? RING_B : SLAB_END));
    auto issue_bias = [&](int tn_) {
        if constexpr (PERSIST) {
            static_assert(BN % 64 == 0 && BN / 64 <= NW, "one 64-float piece per wavefront");
            if (wave < BN / 64)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rBias,
                    (__attribute__((address_space(3))) void*)(bias_lds + wave * 64), 4,
                    (int)((tn_ * BN + wave * 64 + lane) * 4), 0, 0, 0);
        }
    };
    // per-lane LDS element offsets of the fragments (row part; the chunk is XORed per k-step)
    int offA[TI], offB[TJ], swA[TI], swB[TJ];
#pragma unroll
    for (int i = 0; i < TI; ++i) {
        const int r = wm * WM + i * 32 + lr;
        offA[i] = r * BKD;
        swA[i] = (r >> SH) & (CPR - 1);
    }
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
        const int r = wn * WN + j * 32 + lr;
        offB[j] = BM * BKD + r * BKD;
        swB[j] = (r >> SH) & (CPR - 1);
    }
    auto frag = [&](int kt, int ks, bf16x8 (&xa)[TI], bf16x8 (&xb)[TJ]) {
        const uint16_t* st = sm + (kt % S) * STAGE;
        const int c = ks * 2 + hl;
#pragma unroll
        for (int i = 0; i < TI; ++i) xa[i] = *(const bf16x8*)(st + offA[i] + (c ^ swA[i]) * 8);
#pragma unroll
        for (int j = 0; j < TJ; ++j) xb[j] = *(const bf16x8*)(st + offB[j] + (c ^ swB[j]) * 8);
    };

    f32x16 acc[TI][TJ];
    const int nk = K / BKD;
#pragma unroll
    for (int p = 0; p < S - 1; ++p)
        if (p < nk) issue(p);
    issue_bias(tn);
    wait_vm<0>();
    bare_barrier();
    bf16x8 fa[2][TI], fb[2][TJ];
    // one k-slice: MFMAs on the fragments in hand while the next fragments are read.  NEXT:
    // whether the following slice's first fragments are read at the end (after its barrier);
    // WAITN: vmcnt that guarantees the following slice has landed.  The three uses below are
    // separate instantiations, so the steady-state loop body has no branch.
    auto mfmas = [&](int cur, int from, int to) {
#pragma unroll
        for (int q = from; q < to; ++q) {
            const int i = q / TJ, j = q % TJ;
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[cur][j], fa[cur][i], acc[i][j],
                                                                0, 0, 0);
        }
    };
    // Interleave for one k-step (in-order issue: a read placed after a run of MFMAs would wait
    // for the MFMA pipe): reads of the next fragments go between the MFMAs of this k-step.
    constexpr int NM = TI * TJ, NR = TI + TJ;      // MFMAs and fragment reads per k-step
    constexpr int PAIRS = NR < NM ? NR : NM;
    constexpr int PRE = NM / 4;                    // MFMAs issued before a stage barrier
    constexpr int PAIRS2 = NR < NM - PRE ? NR : NM - PRE;
    auto slice = [&](int kt, auto next, auto waitn) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int cur = ks & 1;
            if (ks + 1 < KS) {
                frag(kt, ks + 1, fa[cur ^ 1], fb[cur ^ 1]);
                mfmas(cur, 0, NM);
#pragma unroll
                for (int q = 0; q < PAIRS; ++q) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read
                }
                if constexpr (NR > PAIRS) __builtin_amdgcn_sched_group_barrier(0x100, NR - PAIRS, 0);
                if constexpr (NM > PAIRS) __builtin_amdgcn_sched_group_barrier(0x008, NM - PAIRS, 0);
                __builtin_amdgcn_sched_barrier(0);
            } else if constexpr (decltype(next)::value) {
                mfmas(cur, 0, PRE);
                __builtin_amdgcn_sched_barrier(0);
                wait_vm<decltype(waitn)::value>();
                bare_barrier();
                frag(kt + 1, 0, fa[cur ^ 1], fb[cur ^ 1]);
                mfmas(cur, PRE, NM);
#pragma unroll
                for (int q = 0; q < PAIRS2; ++q) {
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                }
                if constexpr (NR > PAIRS2) __builtin_amdgcn_sched_group_barrier(0x100, NR - PAIRS2, 0);
                if constexpr (NM - PRE > PAIRS2) __builtin_amdgcn_sched_group_barrier(0x008, NM - PRE - PAIRS2, 0);
                __builtin_amdgcn_sched_barrier(0);
            } else {
                mfmas(cur, 0, NM);
            }
        }
    };
    using T_ = std::integral_constant<bool, true>;
    using F_ = std::integral_constant<bool, false>;
    for (;;) {   // one tile; persistent head blocks go on to tile bid + stride
        // the accumulators start at the bias of their column (lane l, register r of MFMA tile j:
        // column (r/4)*8 + (l/32)*4 + r%4 of the tile), so the epilogue does not add it
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
            f32x16 b;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int bc = wn * WN + j * 32 + g * 8 + hl * 4;
                const f32x4 v = PERSIST ? *(const f32x4*)(bias_lds + bc)
                                        : *(const f32x4*)(a.bias + tn * BN + bc);
#pragma unroll
                for (int e = 0; e < 4; ++e) b[g * 4 + e] = v[e];
            }
#pragma unroll
            for (int i = 0; i < TI; ++i) acc[i][j] = b;
        }

        frag(0, 0, fa[0], fb[0]);
        int kt = 0;
        for (; kt + S - 1 < nk; ++kt) {   // steady state: a new slice enters the ring every step
            issue(kt + S - 1);            // slot of slice kt-1: every wave read it before a barrier
            slice(kt, T_(), std::integral_constant<int, (S - 2) * L>());
        }
        for (; kt + 1 < nk; ++kt) slice(kt, T_(), std::integral_constant<int, 0>());   // drain
        // persistent: the block's next tile takes its first slice into slot 0 now -- every wave
        // finished reading slot 0 (slice nk - 2) before the last barrier -- so that it lands while
        // this tile's last slice and epilogue run
        const int nbid = bid + stride;
        const bool more = PERSIST && S == 2 && nk % 2 == 0 && nbid < active;
        int ntm = 0, ntn = 0;
        if (more) {
            setup(nbid, ntm, ntn);
            issue(0);
            issue_bias(ntn);
        }
        slice(kt, F_(), std::integral_constant<int, 0>());   // last slice

        __syncthreads();   // every wave is done with the LDS ring
        // (persistent: the slabs sit past slot 0, which holds the next tile's first slice)
        float* const slabs = (float*)(PERSIST ? sm + STAGE : sm);
        epilogue_lds<E, TI, TJ>(a, acc, slabs + wave * (32 * (TJ * 32 + 4)),
                                m0 + tm * BM + wm * WM, tn * BN + wn * WN, M, lane);
        if (!more) break;
        bid = nbid;
        tm = ntm;
        tn = ntn;
        // the next tile's first slice and bias have landed -- every epilogue issues at least its
        // TI * NQ stores after their copies, and the stores need not be waited for -- and every
        // wave is done with its slab
        wait_vm<TI * (32 / (64 / (TJ * 8)))>();
        bare_barrier();
    }
}

// LDS of one block tile: the DMA ring, reused by the epilogue's per-wave slabs
template <int BM, int BN, int BKD, int S, int WGM, int WGN>
constexpr size_t pipe_lds_bytes() {
    constexpr size_t ring = (size_t)S * (BM + BN) * BKD * 2;
    constexpr size_t slabs = (size_t)WGM * WGN * 32 * (BN / WGN + 4) * 4;
    return ring > slabs ? ring : slabs;
}

// Tail tiles of a split launch: 64 x 64, 64-deep k-slices in a 4-stage ring (three in flight: a
// tail tile is bound by the latency of its k-loop, so few barriers and deep prefetch pay; 32-deep
// slices in 3 or 8 stages measured slower), one per group of four wavefronts.
constexpr int TBM = 64, TBN = 64, TBK = 64, TS = 4;
constexpr size_t TAIL_LDS = pipe_lds_bytes<TBM, TBN, TBK, TS, 2, 2>();
// Middle tail tiles (a partial round of a quarter to half of the grid): 128 x 128, a 2-stage
// ring of 64-deep slices, one per group of four wavefronts.
constexpr int MBM = 128, MBN = 128, MBK = 64, MS = 2;
constexpr size_t MID_LDS = pipe_lds_bytes<MBM, MBN, MBK, MS, 2, 2>();

// Block tiles BM x BN of WGM x WGN wavefronts.  With a.slots set, the launch is split: the
// a.head_grid blocks below it (at most one per slot) are persistent and take the tiles of the
// rows [0, head) that fill whole rounds of the grid (gemm_head_rows) -- tile bid, bid +
// head_grid, ... -- each tile's first k-slice and bias arriving during the previous tile's
// epilogue; the blocks after them cut the remaining rows into 64 x 64 tiles (a partial round of
// at most a quarter of the grid) or 128 x 128 tiles (at most half, with a.mid_tail), one per
// group of four wavefronts, so that the last, partial round spreads over many compute units.
// A tile's outputs are the same whichever block takes it (one k order per output).
template <Epi E, int BM, int BN, int BKD, int S, int WPE, int WGM, int WGN>
__global__ __launch_bounds__(WGM * WGN * 64) __attribute__((amdgpu_waves_per_eu(WPE, WPE)))
void gemm_bf16_pipe_k(GemmArgs a) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    constexpr int NW = WGM * WGN;
    const int wave = threadIdx.x >> 6;
    const int M = a.Mdev ? *a.Mdev : a.Mconst;
    if (!a.slots) {
        pipe_tile<E, BM, BN, BKD, S, WGM, WGN>(a, (uint16_t*)smem, blockIdx.x, 0, M, wave);
        return;
    }
    int kind = 0;
    const int head = gemm_head_rows(M, a.Nout, BM, BN, a.slots, &kind, a.mid_tail);
    if ((int)blockIdx.x < a.head_grid) {
        pipe_tile<E, BM, BN, BKD, S, WGM, WGN, true>(a, (uint16_t*)smem, blockIdx.x, 0, head, wave,
                                                     a.head_grid);
        return;
    }
    static_assert(NW % 4 == 0, "tail tiles take groups of four wavefronts");
    const int grp = wave / 4;
    const int tb = ((int)blockIdx.x - a.head_grid) * (NW / 4) + grp;
    if (kind == 2)
        pipe_tile<E, MBM, MBN, MBK, MS, 2, 2>(a, (uint16_t*)(smem + grp * MID_LDS), tb, head, M,
                                             wave % 4);
    else
        pipe_tile<E, TBM, TBN, TBK, TS, 2, 2>(a, (uint16_t*)(smem + grp * TAIL_LDS), tb, head, M,
                                             wave % 4);
}

template <Epi E, int BM, int BN, int BKD, int S, int WPE, int WGM, int WGN>
constexpr size_t pipe_kernel_lds() {
    constexpr size_t t0 = pipe_lds_bytes<BM, BN, BKD, S, WGM, WGN>();
    constexpr size_t ring_b = (size_t)S * (BM + BN) * BKD * 2;
    constexpr size_t slab_end =
        (size_t)(BM + BN) * BKD * 2 + (size_t)WGM * WGN * 32 * (BN / WGN + 4) * 4;
    constexpr size_t tp = (ring_b > slab_end ? ring_b : slab_end) + (size_t)BN * 4;
    constexpr size_t t = t0 > tp ? t0 : tp;
    constexpr size_t tail = (TAIL_LDS > MID_LDS ? TAIL_LDS : MID_LDS) * (WGM * WGN / 4);
    return t > tail ? t : tail;
}

// Blocks of this configuration that fit on one compute unit (0 if the query fails).
template <Epi E, int BM, int BN, int BKD, int S, int WPE, int WGM, int WGN>
int pipe_blocks_per_cu(const void* k, size_t lds) {
    static int n = -1;
    if (n < 0) {
        int v = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&v, k, WGM * WGN * 64, lds) != hipSuccess)
            v = 0;
        n = v;
    }
    return n;
}

// split: cut the last partial round into 64 x 64 tiles (needs a.cus and Nout % 64 == 0)
template <Epi E, int BM, int BN, int BKD, int S, int WPE, int WGM = 2, int WGN = 2>
void launch_pipe(const GemmArgs& a0, hipStream_t s, bool split = true) {
    static bool raised = false;
    constexpr size_t lds = pipe_kernel_lds<E, BM, BN, BKD, S, WPE, WGM, WGN>();
    static_assert(lds <= 160 * 1024, "LDS exceeds 160 KiB");
    auto k = gemm_bf16_pipe_k<E, BM, BN, BKD, S, WPE, WGM, WGN>;
    if (!raised) {
        (void)hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize,
                                  (int)lds);
        raised = true;
    }
    GemmArgs a = a0;
    const int tn = a.Nout / BN;
    a.head_grid = ((a.Mmax + BM - 1) / BM) * tn;
    a.slots = 0;
    int grid = a.head_grid;
    const int per_cu = split && a.cus > 0 && a.Nout % TBN == 0
                           ? pipe_blocks_per_cu<E, BM, BN, BKD, S, WPE, WGM, WGN>((const void*)k, lds)
                           : 0;
    if (per_cu > 0) {
        a.slots = a.cus * per_cu;
        // persistent head blocks where tiles can follow one another (a 2-stage ring and an even
        // number of k-slices: pipe_tile's `more`); their number is a multiple of the 8 XCDs, so
        // that tile bid + k * head_grid lands on the XCD tile_coords assigns it.  Otherwise one
        // block per head tile, as each block then takes a single tile.
        if (S == 2 && (a.K / BKD) % 2 == 0) a.head_grid = std::min(a.head_grid, a.slots);
        grid = a.head_grid;
        // 128 x 128 tiles for a partial round of a quarter to half of the grid where the output
        // has at most four large tile columns (FC2, out-projection): ViT-B/16 (64 frames) FC2
        // 1.05 -> 0.84 ms, out-projection 0.39 -> 0.33 ms per sweep, ViT-L/14 FC2 -2.4 %;
        // the wider outputs, whose partial rounds are a smaller share, measured 0.5 % slower
        a.mid_tail = a.Nout % MBN == 0 && tn <= 4;
        // the tail holds at most a quarter round of large tiles in 64 x 64 tiles (slots/4/tn
        // tile rows) or at most half a round in 128 x 128 tiles
        const int rows64 = std::min(a.Mmax, (a.slots / 4 / tn + 1) * BM);
        const int tiles64 = ((rows64 + TBM - 1) / TBM) * (a.Nout / TBN);
        const int rows128 = std::min(a.Mmax, (a.slots / 2 / tn + 1) * BM);
        const int tiles128 = a.mid_tail ? ((rows128 + MBM - 1) / MBM) * (a.Nout / MBN) : 0;
        constexpr int per_block = WGM * WGN / 4;
        grid += (std::max(tiles64, tiles128) + per_block - 1) / per_block;
    }
    if (grid > 0) hipLaunchKernelGGL(k, dim3(grid), dim3(WGM * WGN * 64), lds, s, a);
}

// ---------------- fp32 VALU GEMM: block tile 64 x 64, k-step 16, 4 x 4 outputs per thread ---
constexpr int FBM = 64, FBN = 64, FBK = 16;

template <Epi E>
__global__ __launch_bounds__(256) void gemm_f32_k(GemmArgs a) {
    __shared__ float sA[FBK][FBM + 4];
    __shared__ float sB[FBK][FBN + 4];
    const int M = a.Mdev ? *a.Mdev : a.Mconst;
    const int tilesN = a.Nout / FBN;
    const int tm = blockIdx.x / tilesN, tn = blockIdx.x % tilesN;
    if (tm * FBM >= M) return;
    const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
    const int K = a.K;
    const float* A = (const float*)a.A;
    const float* W = (const float*)a.W;
    float acc[4][4] = {};
    for (int k0 = 0; k0 < K; k0 += FBK) {
        // 64 rows x 16 k of A and of W: 1024 values each, 4 per thread
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int e = tid + 256 * t;
            const int rr = e / FBK, kk = e % FBK;
            const int grow = tm * FBM + rr;
            const int arow = a.a_idx ? (grow < M ? a.a_idx[grow] : 0) : grow;
            sA[kk][rr] = A[(size_t)arow * K + k0 + kk];
            sB[kk][rr] = W[(size_t)(tn * FBN + rr) * K + k0 + kk];
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < FBK; ++kk) {
            float av[4], bv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) av[i] = sA[kk][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) bv[j] = sB[kk][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = tm * FBM + ty * 4 + i;
        if (row >= M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) epi_store<E, false>(a, row, tn * FBN + tx * 4 + j, acc[i][j]);
    }
}


// Tile configuration: 0 the choice in launch_one; tuning overrides (DV_GEMM_CFG): 1 = 256 x 128
// everywhere, 3 = without the split last round.
int gemm_cfg() {
    static int v = -1;
    if (v < 0) {
        const char* e = getenv("DV_GEMM_CFG");
        v = e ? atoi(e) : 0;
    }
    return v;
}

template <Epi E>
void launch_one(bool bf16, const GemmArgs& a, hipStream_t s) {
    if (!bf16) {
        const int grid = ((a.Mmax + FBM - 1) / FBM) * (a.Nout / FBN);
        hipLaunchKernelGGL(gemm_f32_k<E>, dim3(grid), dim3(256), 0, s, a);
        return;
    }
    // 256 x 256 tiles of eight wavefronts with a double-buffered 64-deep k-slice (one block per
    // CU) wherever Nout allows, else 256 x 128 tiles, two blocks per CU
    const bool wide = a.Nout % 256 == 0;
    const int cfg = gemm_cfg();
    const bool big = cfg != 1 && wide;
    const bool split = cfg != 3;
    if (big) launch_pipe<E, 256, 256, 64, 2, 2, 2, 4>(a, s, split);
    else launch_pipe<E, 256, 128, 32, 3, 2>(a, s, split);
}

}  // namespace

void launch_gemm(Epi e, bool bf16, const GemmArgs& a, hipStream_t s) {
    switch (e) {
        case Epi::Patch: launch_one<Epi::Patch>(bf16, a, s); break;
        case Epi::Qkv: launch_one<Epi::Qkv>(bf16, a, s); break;
        case Epi::OProj: launch_one<Epi::OProj>(bf16, a, s); break;
        case Epi::Fc1: launch_one<Epi::Fc1>(bf16, a, s); break;
        case Epi::Fc2: launch_one<Epi::Fc2>(bf16, a, s); break;
        case Epi::Restore: launch_one<Epi::Restore>(bf16, a, s); break;
        case Epi::Delta: launch_one<Epi::Delta>(bf16, a, s); break;
    }
}

}  // namespace dv
