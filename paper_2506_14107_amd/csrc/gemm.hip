// Packed-row GEMMs: C[M, Nout] = A[M, K] * W[Nout, K]^T + fused epilogue.
//
// bf16 path: MFMA v_mfma_f32_32x32x16_bf16 (fp32 accumulate) on LDS-staged tiles.
// Both operands are K-contiguous rows, so A and B fragments are the same kind of
// 16-byte LDS read: lane l takes row (l % 32) and k-slice (l / 32) * 8 .. +8.
// The accumulator of lane l, register j holds row (j/4)*8 + (l/32)*4 + j%4, column l%32.
//
// fp32 path: a plain LDS-tiled VALU GEMM (used by fp32 models).
//
// M (the number of packed recompute rows) lives in device memory; the grid is sized for
// the largest possible M and row tiles past M return at once.
#include "dv_internal.h"

namespace dv {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ inline float gelu_erf(float v) { return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f)); }

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
    } else {  // Fc2
        v += a.resid[(size_t)row * a.Nout + col];
        ((float*)a.out)[(size_t)a.idx[row] * a.Nout + col] = v;
    }
}

// ---------------- bf16 MFMA GEMM: block tile 128 x 128, k-step 32, 4 waves of 64 x 64 --------
constexpr int BM = 128, BN = 128, BK = 32;
constexpr int LDK = BK + 8;  // padded LDS row (bf16 elements): 80 bytes, conflict-free b128 reads

template <Epi E>
__global__ __launch_bounds__(256) void gemm_bf16_k(GemmArgs a) {
    __shared__ __attribute__((aligned(16))) uint16_t sA[BM * LDK];
    __shared__ __attribute__((aligned(16))) uint16_t sB[BN * LDK];
    const int M = a.Mdev ? *a.Mdev : a.Mconst;
    const int tilesN = a.Nout / BN;
    const int tm = blockIdx.x / tilesN, tn = blockIdx.x % tilesN;
    if (tm * BM >= M) return;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int K = a.K;
    const uint16_t* Ab = (const uint16_t*)a.A + (size_t)tm * BM * K;
    const uint16_t* Wb = (const uint16_t*)a.W + (size_t)tn * BN * K;

    // each thread moves 2 16-byte chunks of A and 2 of B per k-step
    int lrow[2], lk[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int c = tid + 256 * i;
        lrow[i] = c >> 2;
        lk[i] = (c & 3) * 8;
    }
    uint4 ra[2], rb[2];
    auto gload = [&](int k0) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            ra[i] = *(const uint4*)(Ab + (size_t)lrow[i] * K + k0 + lk[i]);
            rb[i] = *(const uint4*)(Wb + (size_t)lrow[i] * K + k0 + lk[i]);
        }
    };

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    gload(0);
    for (int k0 = 0; k0 < K; k0 += BK) {
        __syncthreads();
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            *(uint4*)(sA + lrow[i] * LDK + lk[i]) = ra[i];
            *(uint4*)(sB + lrow[i] * LDK + lk[i]) = rb[i];
        }
        __syncthreads();
        if (k0 + BK < K) gload(k0 + BK);
#pragma unroll
        for (int ks = 0; ks < BK; ks += 16) {
            bf16x8 fa[2], fb[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int row = wm * 64 + i * 32 + (lane & 31);
                fa[i] = *(const bf16x8*)(sA + row * LDK + ks + (lane >> 5) * 8);
            }
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int row = wn * 64 + j * 32 + (lane & 31);
                fb[j] = *(const bf16x8*)(sB + row * LDK + ks + (lane >> 5) * 8);
            }
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
        }
    }

#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = tm * BM + wm * 64 + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                const int col = tn * BN + wn * 64 + j * 32 + (lane & 31);
                if (row < M) epi_store<E, true>(a, row, col, acc[i][j][r]);
            }
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
            sA[kk][rr] = A[(size_t)(tm * FBM + rr) * K + k0 + kk];
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

template <Epi E>
void launch_one(bool bf16, const GemmArgs& a, hipStream_t s) {
    if (bf16) {
        const int grid = ((a.Mmax + BM - 1) / BM) * (a.Nout / BN);
        hipLaunchKernelGGL(gemm_bf16_k<E>, dim3(grid), dim3(256), 0, s, a);
    } else {
        const int grid = ((a.Mmax + FBM - 1) / FBM) * (a.Nout / FBN);
        hipLaunchKernelGGL(gemm_f32_k<E>, dim3(grid), dim3(256), 0, s, a);
    }
}

}  // namespace

void launch_gemm(Epi e, bool bf16, const GemmArgs& a, hipStream_t s) {
    switch (e) {
        case Epi::Patch: launch_one<Epi::Patch>(bf16, a, s); break;
        case Epi::Qkv: launch_one<Epi::Qkv>(bf16, a, s); break;
        case Epi::OProj: launch_one<Epi::OProj>(bf16, a, s); break;
        case Epi::Fc1: launch_one<Epi::Fc1>(bf16, a, s); break;
        case Epi::Fc2: launch_one<Epi::Fc2>(bf16, a, s); break;
    }
}

}  // namespace dv
