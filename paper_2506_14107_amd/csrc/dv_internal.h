// Internal interface between the orchestrator (api.hip) and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace dv {

// ---- bf16 storage helpers (raw 16-bit patterns) ---------------------------------------------
__host__ __device__ inline uint16_t f32_to_bf16(float f) {
    uint32_t u = __builtin_bit_cast(uint32_t, f);
    u += 0x7FFFu + ((u >> 16) & 1u);  // round to nearest, ties to even (finite inputs)
    return (uint16_t)(u >> 16);
}
__host__ __device__ inline float bf16_to_f32(uint16_t h) {
    return __builtin_bit_cast(float, (uint32_t)h << 16);
}

// ---- placement of a group's frames on one XCD -------------------------------------------------
// Workgroups are dealt to the 8 XCDs round-robin (block b runs on XCD b % 8), and each XCD has
// its own L2.  A unit of G work items that read the same reference-frame rows (the G frames of
// one group, one head) is placed on one XCD: units u = x, x + 8, ... on XCD x.  Slots for
// `units` units of G items each, in whole rounds of 8:
inline int xcd_unit_grid(int units, int G) { return (units + 7) / 8 * 8 * G; }

// ---- reordered referencing (I/P/B frames with past and future references) --------------------
// Groups of G frames (G a multiple of 4) start with an I frame, computed in full.  Positions
// 4, 8, ... of a group are P frames referencing the anchor four frames back.  Between two
// anchors a and a + 4 (the next group's I frame closes the group's last block) the frame at
// a + 2 is B_dist2, referencing both anchors, and those at a + 1 and a + 3 are B_dist1,
// referencing their neighbours among a, a + 2, a + 4.  A reference at or past frame F (the
// end of the frames at hand) is absent (-1).  type: 0 I, 1 P, 2 B_dist2, 3 B_dist1.
struct FrameRefs {
    int type, past, fut;
};
__host__ __device__ inline FrameRefs reorder_refs(int f, int G, int F) {
    const int p = f % G;
    if (p == 0) return {0, -1, -1};
    const int d = p & 3, a = f - d;
    FrameRefs q;
    if (d == 0) q = {1, f - 4, -1};
    else if (d == 2) q = {2, a, a + 4};
    else if (d == 1) q = {3, a, a + 2};
    else q = {3, a + 2, a + 4};
    if (q.fut >= F) q.fut = -1;
    return q;
}

// ---- GEMM ------------------------------------------------------------------------------------
// C[M, Nout] = A[M, K] * W[Nout, K]^T with a fused epilogue.  M is read on the device.
enum class Epi : int {
    Patch = 0,  // x[(r/P)*N + 1 + r%P, c] = acc + bias[c] + pos[(1 + r%P), c]        (fp32 out)
    Qkv = 1,    // qkv[r, c] = acc + bias[c]                                           (elem out)
    OProj = 2,  // z[r, c] = acc + bias[c] + x[idx[r], c]                              (fp32 out)
    Fc1 = 3,    // h[r, c] = gelu(acc + bias[c])                                       (elem out)
    Fc2 = 4,    // x[idx[r], c] = acc + bias[c] + z[r, c]                              (fp32 out)
    Restore = 5,  // x[t, c] = acc + bias[c] + x[ref(t), c], t = idx[r]: a reused token's row
                  // from its reference token's new row (ref(t): same token of frame G*floor(f/G))
    Delta = 6,    // out[r, c] = acc + bias[c]                                        (fp32 out)
};

struct GemmArgs {
    const void* A;       // [rows, K] row-major; rows padded to the tile height
    const void* W;       // [Nout, K] row-major
    const float* bias;   // [Nout]
    int K, Nout;
    const int* Mdev;     // device row count (nullptr: use Mconst)
    int Mconst;
    int Mmax;            // upper bound on M (grid sizing)
    void* out;
    const float* resid;  // OProj: x rows; Fc2: z rows
    const int* idx;      // packed row -> token row
    const int* a_idx;    // A row gather: packed row m reads A row a_idx[m] (nullptr: row m)
    const float* pos;    // Patch: position table [N, D]
    int P, N;            // Patch: patches and tokens per frame (Restore: N)
    int G;               // Restore: group size
    int cus;             // compute units of the device (0: no split of the last round)
    // set by the launcher: the blocks below head_grid (persistent, at most one per slot) run
    // large tiles over the rows [0, head), the others small tiles over [head, M),
    // head = gemm_head_rows(M, Nout, BM, BN, slots);
    // slots = 0: one tiling for all rows
    int slots, head_grid;
    bool mid_tail;       // a partial round of a quarter to half of the grid goes to 128 x 128 tiles
};

// Rows that large tiles take when the M rows are split between large tiles (hbm x hbn, `slots`
// resident blocks) and small ones: the tile rows that fill whole rounds of the large-tile grid.
// *kind: 1 for a remainder of at most a quarter of a round (64 x 64 tiles), 2 for at most half
// a round when `mid` (128 x 128 tiles), 0 when every row stays in large tiles (no remainder, or
// a larger one).  Each output is the same dot product in the same k order in any tiling, so the
// split does not change results.
__host__ __device__ inline int gemm_head_rows(int M, int Nout, int hbm, int hbn, int slots,
                                              int* kind = nullptr, bool mid = false) {
    const int tn = Nout / hbn;
    const int mt = (M + hbm - 1) / hbm;
    const int mA = (mt * tn / slots) * slots / tn;   // whole tile rows inside the full rounds
    const int rem = (mt - mA) * tn;                  // large tiles of the partial round
    int k = 0;
    if (mA < mt) k = rem * 4 <= slots ? 1 : (mid && rem * 2 <= slots) ? 2 : 0;
    if (kind) *kind = k;
    return k ? mA * hbm : M;
}

void launch_gemm(Epi e, bool bf16, const GemmArgs& a, hipStream_t s);
// Measurement probe: `blocks` blocks of 256 threads run `iters` rounds of four independent bf16
// MFMA chains; returns the FLOPs the launch performs.  sink: blocks*256 floats.
double launch_mfma_loop(int blocks, int iters, float* sink, hipStream_t s);

// ---- attention -------------------------------------------------------------------------------
struct AttnArgs {
    const void* qkv;   // packed rows [M, 3D] (Q | K | V), elem
    const int* pos;    // [F*N] packed row of each token's K/V (reused -> reference's row)
    const int* qoff;   // [F+1] packed query rows of frame f: qoff[f] .. qoff[f+1]
    void* out;         // [M, D] elem
    int F, N, D, H;
    int G;             // group size, 0 without reuse (block placement only)
    int cus;           // compute units of the device (0: one block per work item)
    int skip;          // leading frames carried over from an earlier call (no rows, no queries)
    int sparse;        // reuse on with G == 0: frames hold few query tiles (per-tile wavefronts)
    int tile_cut;      // set by launch_attention: frames with at most this many query tiles go to
                       // per-tile wavefronts, the others to per-frame blocks
};
void launch_attention(bool bf16, const AttnArgs& a, hipStream_t s);
// Class-token attention weights of every non-reference frame (G > 0: frames f % G == 0 are
// skipped), per head: probs[(f*H + h)*N + j] = softmax_j(q_h . k_h,j / sqrt(dh)) with q the
// frame's class-token query (its first packed row, qoff[f]) and k_j its key row through pos.
void launch_cls_attention(bool bf16, const AttnArgs& a, float* probs, hipStream_t s);
size_t attention_lds_bytes(bool bf16, int N, int dh);
bool attention_supported(bool bf16, int N, int dh);

// ---- row kernels -----------------------------------------------------------------------------
void launch_im2col(bool bf16, const float* frames, int F, int S, int p, int Kp, void* A,
                   hipStream_t s);
void launch_cls_init(float* x, const float* cls, const float* pos, int F, int N, int D,
                     hipStream_t s);

enum GateMode : int { GATE_COS = 0, GATE_INJECT = 1, GATE_ALL = 2, GATE_NONE = 3 };
struct GateArgs {
    float* x;             // [F*N, D] (written only to give a recomputed alias its row)
    int F, N, D, G, L, layer;
    int mode;
    float tau;
    const uint8_t* prev;  // previous layer's map (gate mode, monotone shortcut) or nullptr
    const uint8_t* inj;   // injected maps [F, L, N] (batch base) or nullptr
    uint8_t* cur;         // [F*N] this layer's map (or nullptr)
    uint8_t* out_masks;   // [F, L, N] (batch base) or nullptr
    int* cnt;             // [F * gate_chunks(N)] recomputed tokens per block (or nullptr)
    const float* ln_g;    // LN1 gain / shift
    const float* ln_b;
    void* ln_out;         // [F*N, D] elem: LN1 rows of recomputed tokens (token-indexed) or nullptr
    void* d_out;          // [F*N, D] elem: x_f - x_ref rows of reused tokens (token-indexed;
                          // restoration) or nullptr.  May be ln_out: the rows are disjoint.
    const float* dec;     // GATE_COS with the decision MLP: the layer's W_d1 [64,6], b_d1 [64],
                          // W_d2 [64], b_d2 [1] (fp32, back to back), else nullptr
    const float* tcls;    // [F, H, N] class-token attention weights of the previous layer, per
                          // head (nullptr: 1/N); the cue is their mean over the H heads
    int H;
    int reorder;          // reordered referencing (reorder_refs) instead of the star
    uint8_t* src;         // [F*N] reordered: 1 where the future reference supplies the token
    const int* root;      // [F*N] reordered: the previous layer's root map (nullptr: every token
                          // holds its own row); a recomputed token gets its root's row copied in
    int skip;             // leading frames carried over from an earlier call of a stream: one is
                          // the cached reference (the first in the star, the last under
                          // reordering; its rows already in x), the others gaps; none is gated,
                          // and inj / out_masks start at frame skip
};
// Reordering with restoration: a reused row is built along its chain of sources; a group of G
// frames has chains of at most G/4 + 1 reused links (B_dist1, B_dist2, then the P frames back
// to the I frame), so G <= 4 * (CHAIN_MAX - 1).
constexpr int CHAIN_MAX = 16;
constexpr int DEC_HIDDEN = 64;   // decision MLP hidden units: one per lane of a wavefront
constexpr int DEC_FEAT = 6;      // its features: s, t, one-hot type (I, P, B_dist2, B_dist1)
constexpr int DEC_FLOATS = DEC_HIDDEN * DEC_FEAT + 2 * DEC_HIDDEN + 1;
// Mode GATE_NONE marks every token recomputed (reuse off) and only writes LN1 rows.
// The gate runs in blocks of GATE_TOK tokens; counts are per block: cnt[f * gate_chunks(N) + c].
constexpr int GATE_TOK = 16;
inline int gate_chunks(int N) { return (N + GATE_TOK - 1) / GATE_TOK; }
void launch_gate(bool bf16, const GateArgs& a, hipStream_t s);
void launch_count(const uint8_t* m, int F, int N, int G, int* cnt, hipStream_t s);
// qoff[0..F] = exclusive prefix of the per-frame counts (sum of `per` consecutive entries of
// cnt per frame), M[0] = qoff[F]; M[1] = tokens - M[0] (the reused tokens) when tokens > 0
void launch_scan(const int* cnt, int per, int F, int tokens, int* qoff, int* M, hipStream_t s);
// idx/pos from a per-layer map and its qoff (cur == nullptr: every token recomputed, identity
// lists, qoff_in ignored and qoff_out written)
// ridx (or nullptr): the reused tokens f*N+i of non-reference frames in frame-major order, at
// slot (f*N - qoff[f]) + (reused tokens of frame f before i)
// skip > 0 (stream): frames below skip have no rows; one of them is the cached reference (the
// first in the star, the last under reordering), whose keys and values sit at packed rows
// ext_row .. ext_row + N - 1: pos of every token of those frames points there
// rslot (or nullptr): for every reused token, its slot in ridx
void launch_compact(const uint8_t* cur, const int* qoff_in, int F, int N, int G, int* idx,
                    int* pos, int* qoff_out, int* ridx, hipStream_t s, int skip = 0,
                    int ext_row = 0, int* rslot = nullptr);
// launch_scan then launch_compact in one launch: every block sums the per-block counts of the
// frames before it (and before its reference) itself; qoff, M as launch_scan writes them
void launch_scan_compact(const int* cnt, int per, int tokens, const uint8_t* cur, int F, int N,
                         int G, int* idx, int* pos, int* qoff, int* M, int* ridx, hipStream_t s,
                         int skip = 0, int ext_row = 0, int* rslot = nullptr);
// dst[i, 0:2D] = K|V of packed row pos[f*N + i], el-byte elems
void launch_copy_ref_kv(const void* qkv, const int* pos, int f, int N, int D, int el, void* dst,
                        hipStream_t s);
// dst[i, 0:D] = x row of token i of frame root[f*N + i] (root == nullptr: of frame f)
void launch_copy_rows(const float* x, const int* root, int f, int N, int D, float* dst,
                      hipStream_t s);

// LayerNorm of rows (optionally gathered through idx) into elem rows: dst[r] = LN(src[g(r)])
void launch_ln_rows(bool bf16, const float* src, const int* gather, const int* Mdev, int Mmax,
                    int D, const float* g, const float* b, void* dst, hipStream_t s);
// x[f*N+i] = x[r*N+i] for every token with cur[f*N+i] != 0, r = root[f*N+i] (root == nullptr:
// the group's first frame)
void launch_merge(float* x, const uint8_t* cur, const int* root, int F, int N, int D, int G,
                  hipStream_t s);
// Reordered referencing with the restoration layer: every reused token's new row, built along its
// chain of sources from the root's new row: x[t] = ((x[root] + d[link_1]) + ...) + d[t], where
// d[u] = rbuf[rslot[u]] is token u's restoration output and the links run from the root outward.
// Mdev: the number of reused tokens (rows of ridx).
void launch_restore_chain(float* x, const float* rbuf, const int* ridx, const int* rslot,
                          const uint8_t* cur, const uint8_t* src, const int* Mdev, int Mmax, int F,
                          int N, int D, int G, hipStream_t s);
// Reordered referencing: for every reused token, follow the sources (src, reorder_refs) to the
// frame r that recomputes it; pos[f*N+i] = pos[r*N+i], root[f*N+i] = r (f for recomputed ones).
void launch_resolve(const uint8_t* cur, const uint8_t* src, int F, int N, int G, int* pos,
                    int* root, hipStream_t s);
// emb[f] = LN(x[f*N]) (class token)
void launch_final_ln(const float* x, int F, int N, int D, const float* g, const float* b,
                     float* emb, hipStream_t s);
void launch_fill_u8(uint8_t* p, size_t n, uint8_t v, hipStream_t s);
// out_masks[f, layer, :] = 0 for all f (dense mode)
void launch_zero_mask_layer(uint8_t* out_masks, int F, int L, int N, int layer, hipStream_t s);

}  // namespace dv
