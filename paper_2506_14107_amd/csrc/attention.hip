// Attention over mixed fresh and reference K/V.
//
// One block per (frame f, head h).  The block stages the frame's N keys and values of
// head h in LDS, reading each key row through pos[]: a recomputed token's own packed row,
// or -- for a reused token -- the packed row of the same token of the reference frame.
// Each wavefront then takes the frame's packed query rows qoff[f] .. qoff[f+1] in turn:
// scores (lane-strided over keys), softmax in fp32 with wave reductions, then P.V with one
// lane per output dimension.
#include "dv_internal.h"

namespace dv {

namespace {

constexpr int NWAVE = 4;

// Orders LDS writes and reads of one wavefront (its lanes exchange data through LDS).
__device__ inline void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ inline float wmax(float v) {
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}
__device__ inline float wsum(float v) {
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

template <bool BF>
struct Lds {
    static constexpr int pad = BF ? 2 : 1;
    typedef typename std::conditional<BF, uint16_t, float>::type T;
};

template <bool BF>
__device__ inline float ld(const void* p, size_t i) {
    if (BF) return bf16_to_f32(((const uint16_t*)p)[i]);
    return ((const float*)p)[i];
}

template <bool BF>
__global__ __launch_bounds__(256) void attn_k(AttnArgs a) {
    typedef typename Lds<BF>::T T;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int f = blockIdx.x, h = blockIdx.y;
    const int N = a.N, D = a.D, dh = D / a.H;
    const int ldk = dh + Lds<BF>::pad;
    T* Ks = (T*)smem;
    T* Vs = Ks + (size_t)N * ldk;
    float* qs = (float*)(((uintptr_t)(Vs + (size_t)N * dh) + 15) & ~(uintptr_t)15);
    float* ps = qs + NWAVE * dh;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const size_t ld3 = 3 * (size_t)D;
    const T* qkv = (const T*)a.qkv;

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
        for (int d = lane; d < dh; d += 64) myq[d] = ld<BF>(qkv, (size_t)q * ld3 + h * dh + d) * scale;
        wave_lds_sync();
        float mx = -INFINITY;
        for (int j = lane; j < N; j += 64) {
            float s = 0.f;
            const T* kr = Ks + j * ldk;
            for (int d = 0; d < dh; ++d) {
                float kv;
                if (BF) kv = bf16_to_f32(((const uint16_t*)kr)[d]);
                else kv = ((const float*)kr)[d];
                s = fmaf(myq[d], kv, s);
            }
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
            for (int j = 0; j < N; ++j) {
                float vv;
                if (BF) vv = bf16_to_f32(((const uint16_t*)Vs)[j * dh + d]);
                else vv = ((const float*)Vs)[j * dh + d];
                o = fmaf(myp[j], vv, o);
            }
            o *= inv;
            if (BF) ((uint16_t*)a.out)[(size_t)q * D + h * dh + d] = f32_to_bf16(o);
            else ((float*)a.out)[(size_t)q * D + h * dh + d] = o;
        }
        wave_lds_sync();  // this wave's myq/myp are rewritten by its next query
    }
}

}  // namespace

size_t attention_lds_bytes(bool bf16, int N, int dh) {
    const size_t el = bf16 ? 2 : 4;
    const size_t ldk = dh + (bf16 ? 2 : 1);
    size_t b = (size_t)N * ldk * el + (size_t)N * dh * el;
    b = (b + 15) & ~(size_t)15;
    return b + (size_t)NWAVE * dh * 4 + (size_t)NWAVE * N * 4;
}

void launch_attention(bool bf16, const AttnArgs& a, hipStream_t s) {
    const int dh = a.D / a.H;
    const size_t lds = attention_lds_bytes(bf16, a.N, dh);
    static bool raised[2] = {false, false};
    if (!raised[bf16]) {  // allow more than the default dynamic LDS (gfx950 has 160 KiB per CU)
        (void)hipFuncSetAttribute(bf16 ? (const void*)attn_k<true> : (const void*)attn_k<false>,
                                  hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        raised[bf16] = true;
    }
    if (bf16) hipLaunchKernelGGL(attn_k<true>, dim3(a.F, a.H), dim3(256), lds, s, a);
    else hipLaunchKernelGGL(attn_k<false>, dim3(a.F, a.H), dim3(256), lds, s, a);
}

}  // namespace dv
