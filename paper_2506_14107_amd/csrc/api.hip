// C ABI and host orchestrator of the reuse-aware ViT encoder.
//
// Per internal batch of whole groups (layer-wise scheduling: one layer over every frame of
// the batch before the next), the launch sequence is
//   im2col -> patch GEMM (+bias +pos) ; class-token rows
//   for each layer:
//     gate (cosine to the reference, or injected map) + per-frame counts
//     compaction (idx / pos / qoff / M, all on the device)
//     LN1 of the gathered recompute rows -> QKV GEMM -> attention over fresh + reference K/V
//     -> out-proj GEMM (+bias, +gathered residual) -> LN2 -> FC1 GEMM (+bias, GELU)
//     -> FC2 GEMM (+bias, +residual) written straight back into the token rows
//     [injection mode: copy the reference's new row into every reused row]
//     [restoration: the gate also writes x_f - x_ref of every reused token, the compaction the
//      reused-token list; a D -> 128 GEMM (+bias, GELU) on those rows runs before QKV and a
//      128 -> D GEMM (+bias, + the reference token's new row) after FC2 writes the reused rows]
//     [decision MLP: the gate evaluates it on (cosine, class-token attention of the previous
//      layer, frame type); after attention the class-token weights of every frame are
//      computed for the next layer]
//     [reordered referencing: the gate compares each token with the frame's past and future
//      anchors and records which one supplies it; after the compaction every reused token's
//      key/value row is resolved along those sources to the frame that recomputes it (its
//      root); a reused token's row stays that frame's new row, read through the root map by the
//      next layer's gate, and is filled in only to hand out tokens.  An internal batch also
//      carries the next batch's first frame (an I frame, the future anchor of its last block).]
//   [stream (dv_stream_encode): a group may span calls.  The reference of a group that is still
//    open when a call ends keeps its per-layer input rows and keys/values in a cache; the next
//    call's first batch starts with that reference as local frame 0 (rows copied from the
//    cache, not recomputed), then gap frames standing for the group's frames of earlier calls,
//    then the call's own frames, so that groups keep their positions (frame f's reference is
//    frame G * floor(f / G) of the batch).  Reordered: the frames after the last anchor are
//    held until it arrives; a batch starts at a group boundary with gap frames up to the cached
//    anchor (their last), then the held and new frames, and ends on an anchor, which is cached.]
//   final LayerNorm of the class tokens.
// Nothing is read back to the host inside an encode call.
//
// Gate mode needs no merge pass: once a token is reused its row would be a copy of the
// reference's, whose cosine is exactly 1, so it stays reused in every later layer; the gate
// answers such tokens from the previous layer's map and nobody reads their rows again.  Only
// when the caller asks for the full token buffer are those rows filled in at the end.  Under
// the decision MLP a reused token may be recomputed later (its other cues change): its cosine
// is still exactly 1, and when the MLP recomputes it the gate first copies the reference's
// row into it.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/dejavu.h"
#include "dv_internal.h"

using namespace dv;

// Scratch of dv_encode_noalloc: the workspace of its internal batches, in a static device array
// (one copy per device, held until the process ends).  Host code never uses the array's name as
// an address: dv_create looks up each device's copy once (scratch_setup) and every launch takes
// that address.
static __device__ __align__(256) char scratch[DV_SCRATCH_BYTES];

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

#define HIP_TRY(expr)                                                                          \
    do {                                                                                       \
        hipError_t e_ = (expr);                                                                \
        if (e_ != hipSuccess)                                                                  \
            return fail(e_ == hipErrorOutOfMemory ? DV_ENOMEM : DV_EHIP, "%s: %s (%s:%d)", #expr, \
                        hipGetErrorString(e_), __FILE__, __LINE__);                            \
    } while (0)

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch[MAX_DEVICES] = {};   // device address of each device's copy of `scratch`
bool g_scratch_done[MAX_DEVICES] = {};
std::string g_scratch_err;           // why a look-up failed

// Once per device, with that device current: the address of its copy of the scratch array,
// cleared once (later calls find the previous call's contents, as in a handle's workspace).
void scratch_setup(int dev) {
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (dev < 0 || dev >= MAX_DEVICES) {
        g_scratch_err = "device index out of range";
        return;
    }
    if (g_scratch_done[dev]) return;
    g_scratch_done[dev] = true;
    void* p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e == hipSuccess) e = hipMemset(p, 0, DV_SCRATCH_BYTES);
    if (e != hipSuccess) {
        g_scratch_err = hipGetErrorString(e);
        return;
    }
    g_scratch[dev] = p;
}

void* scratch_base(int dev) {
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    return (dev >= 0 && dev < MAX_DEVICES) ? g_scratch[dev] : nullptr;
}

constexpr int ROW_PAD = 256;  // GEMM operand rows are padded to a multiple of the tallest tile

size_t round_up(size_t v, size_t m) { return (v + m - 1) / m * m; }

struct LayerW {
    const float *ln1_g, *ln1_b, *b_qkv, *b_o, *ln2_g, *ln2_b, *b_1, *b_2;
    const void *W_qkv, *W_o, *W_1, *W_2;
    const void *W_r1, *W_r2;      // restoration MLP (DV_FLAG_RESTORE), else null
    const float *b_r1, *b_r2;
    const float* dec;             // decision MLP (DV_FLAG_DECISION): DEC_FLOATS fp32, else null
};

struct Dims {
    int S, p, L, D, H, Dm, N, P, Kp, B;
    bool bf16;
    bool restore;   // DV_FLAG_RESTORE
    bool decision;  // DV_FLAG_DECISION
    bool reorder;   // DV_FLAG_REORDER
    int Bw;         // frames of workspace: B, plus one look-ahead frame with reordering
};

constexpr int RH = DV_RESTORE_HIDDEN;

// validates a configuration; fills dims
int check_config(const dv_config* c, Dims* d) {
    if (!c) return fail(DV_EINVAL, "config is NULL");
    if (c->image_size < 1 || c->patch < 1 || c->depth < 1 || c->width < 1 || c->heads < 1 ||
        c->mlp < 1 || c->max_batch_frames < 1)
        return fail(DV_EINVAL, "config sizes must be >= 1");
    if (c->dtype != DV_F32 && c->dtype != DV_BF16) return fail(DV_EINVAL, "unknown dtype %d", c->dtype);
    if (c->flags & ~(DV_FLAG_RESTORE | DV_FLAG_DECISION | DV_FLAG_REORDER))
        return fail(DV_EUNSUPPORTED, "unknown flag bits 0x%x", c->flags);
    if (c->image_size % c->patch) return fail(DV_EUNSUPPORTED, "image_size %% patch != 0");
    if (c->width % c->heads) return fail(DV_EUNSUPPORTED, "width %% heads != 0");
    const int dh = c->width / c->heads;
    if (dh % 16 || dh > 128) return fail(DV_EUNSUPPORTED, "head dim %d must be a multiple of 16, <= 128", dh);
    const bool bf = c->dtype == DV_BF16;
    const int tile = bf ? 128 : 64;
    if (c->width % tile || c->mlp % tile)
        return fail(DV_EUNSUPPORTED, "width and mlp must be multiples of %d for this dtype", tile);
    if (c->width > 2048) return fail(DV_EUNSUPPORTED, "width above 2048");
    d->S = c->image_size;
    d->p = c->patch;
    d->L = c->depth;
    d->D = c->width;
    d->H = c->heads;
    d->Dm = c->mlp;
    const int g = c->image_size / c->patch;
    d->P = g * g;
    d->N = d->P + 1;
    d->Kp = (int)round_up((size_t)3 * c->patch * c->patch, 64);
    d->B = c->max_batch_frames;
    d->bf16 = bf;
    d->restore = (c->flags & DV_FLAG_RESTORE) != 0;
    d->decision = (c->flags & DV_FLAG_DECISION) != 0;
    d->reorder = (c->flags & DV_FLAG_REORDER) != 0;
    d->Bw = d->B + (d->reorder ? 1 : 0);
    if (!attention_supported(bf, d->N, dh))
        return fail(DV_EUNSUPPORTED, "attention for N=%d tokens, head dim %d is not supported "
                    "(bf16: head dim 64/80/96/128; keys and values of a head must fit in LDS)", d->N, dh);
    // kernels address each workspace buffer with 32-bit byte offsets (buffer descriptors) and
    // token rows with int indices: every buffer stays below 2^32 bytes, the qkv rows including
    // a stream's cached reference rows after the batch's
    const size_t T = (size_t)d->Bw * d->N, Tp = round_up(T, ROW_PAD);
    const size_t el = bf ? 2 : 4, D = d->D;
    const size_t bufs[] = {T * D * 4,                                         // x
                           Tp * std::max(D, (size_t)d->Kp) * el,              // A
                           (Tp + round_up(d->N, ROW_PAD)) * 3 * D * el,       // qkv
                           Tp * D * 4,                                        // Z (O is smaller)
                           Tp * (size_t)d->Dm * el,                           // MLP hidden
                           d->restore ? Tp * (size_t)RH * el : 0,             // restoration hidden
                           (d->restore && d->reorder) ? Tp * D * 4 : 0};      // restoration outputs
    size_t largest = 0;
    for (size_t b : bufs) largest = std::max(largest, b);
    if (largest >= (1ull << 32) || T >= (1ull << 30))
        return fail(DV_EUNSUPPORTED, "max_batch_frames %d: a workspace buffer of %zu bytes is "
                    "too large for 32-bit offsets", d->B, largest);
    return DV_OK;
}

size_t blob_floats(const Dims& d) {
    const size_t D = d.D, Dm = d.Dm, N = d.N, p = d.p;
    size_t per_layer = 2 * D + 3 * D * D + 3 * D + D * D + D + 2 * D + Dm * D + Dm + D * Dm + D;
    const size_t restore = d.restore ? (size_t)d.L * (2 * RH * D + RH + D) : 0;
    const size_t decision = d.decision ? (size_t)d.L * DEC_FLOATS : 0;
    return D * 3 * p * p + D + D + N * D + (size_t)d.L * per_layer + 2 * D + restore + decision;
}

// Workspace of one internal batch size: the buffers every launch of an encode reads and writes.
// A handle carves one from its own allocation (with the stream state); dv_encode_noalloc carves
// one from the static scratch array.
struct Work {
    float* x = nullptr;         // [T, D] fp32 token rows
    void* A = nullptr;          // [Tp, max(D, Kp)] elem: LN output / patch rows
    void* qkv = nullptr;        // [Tp (+ Np with the stream state), 3D] elem
    int ext_row = 0;            // packed row of the cached reference's first key/value row
    void* O = nullptr;          // [Tp, D] elem: attention output
    float* Z = nullptr;         // [Tp, D] fp32: after attention residual
    void* Hb = nullptr;         // [Tp, Dm] elem: MLP hidden
    uint8_t* mask[2] = {nullptr, nullptr};   // [T] per-layer maps (ping-pong)
    int *idx = nullptr, *pos_ = nullptr, *qoff = nullptr, *cnt = nullptr;
    int* M = nullptr;           // M[0]: recomputed rows, M[1]: reused tokens
    int *idx_id = nullptr, *pos_id = nullptr, *qoff_id = nullptr;   // identity lists (reuse off)
    int id_frames = -1;         // frames the identity lists were built for
    int* ridx = nullptr;        // [T] reused tokens (restoration)
    void* Hr = nullptr;         // [Tp, 128] elem: restoration hidden rows
    float* tcls = nullptr;      // [Bw, H, N] class-token attention weights per head (decision MLP)
    uint8_t* srcmap = nullptr;  // [T] reordered: 1 where the future anchor supplies the token
    int* root = nullptr;        // [T] reordered: frame that recomputes a reused token
    int* rslot = nullptr;       // [T] reordered restoration: a reused token's slot in ridx
    float* rbuf = nullptr;      // [Tp, D] reordered restoration: restoration outputs
    // stream state (handles only): the cached reference's layer inputs x^0 .. x^L [L+1, N, D]
    // fp32 and keys/values [L, N, 2D] elem; under reordering the held frames' pixels
    // [3, 3, S, S], their maps [3, L, N] and a staging area for a batch's maps [B, L, N]
    float* xc = nullptr;
    void* kvc = nullptr;
    float* hold = nullptr;
    uint8_t* holdm = nullptr;
    uint8_t* injs = nullptr;
};

// The one layout of a workspace for dimensions d (d.Bw frames): returns its bytes and, with a
// base, the views into it.  stream: also the stream state and the spare key/value rows of a
// stream's cached reference.
size_t carve_work(const Dims& d, char* base, Work* out, bool stream) {
    const size_t N = d.N, D = d.D, Dm = d.Dm, L = d.L, el = d.bf16 ? 2 : 4;
    const size_t T = (size_t)d.Bw * N, Tp = round_up(T, ROW_PAD);
    const size_t Awide = std::max((size_t)D, (size_t)d.Kp);
    size_t off = 0;
    auto take = [&](size_t bytes) -> char* {
        char* r = base ? base + off : nullptr;
        off += round_up(bytes, 256);
        return r;
    };
    Work w;
    w.x = (float*)take(T * D * 4);
    w.A = take(Tp * Awide * el);
    w.qkv = take((Tp + (stream ? round_up(N, ROW_PAD) : 0)) * 3 * D * el);
    w.ext_row = (int)Tp;
    w.O = take(Tp * D * el);
    w.Z = (float*)take(Tp * D * 4);
    w.Hb = take(Tp * Dm * el);
    w.mask[0] = (uint8_t*)take(T);
    w.mask[1] = (uint8_t*)take(T);
    w.idx = (int*)take(T * 4);
    w.pos_ = (int*)take(T * 4);
    w.qoff = (int*)take((d.Bw + 1) * 4);
    w.idx_id = (int*)take(T * 4);
    w.pos_id = (int*)take(T * 4);
    w.qoff_id = (int*)take((d.Bw + 1) * 4);
    w.cnt = (int*)take((size_t)d.Bw * gate_chunks(d.N) * 4);
    w.M = (int*)take(4 * 4);
    if (d.restore) {
        w.ridx = (int*)take(T * 4);
        w.Hr = take(Tp * RH * el);
    }
    if (d.decision) w.tcls = (float*)take(T * d.H * 4);
    if (d.reorder) {
        w.srcmap = (uint8_t*)take(T);
        w.root = (int*)take(T * 4);
    }
    if (d.reorder && d.restore) {
        w.rslot = (int*)take(T * 4);
        w.rbuf = (float*)take(Tp * D * 4);
    }
    if (stream) {
        w.xc = (float*)take((L + 1) * N * D * 4);
        w.kvc = take(L * N * 2 * D * el);
        if (d.reorder) {
            w.hold = (float*)take((size_t)3 * 3 * d.S * d.S * 4);
            w.holdm = (uint8_t*)take(3 * L * N);
            w.injs = (uint8_t*)take((size_t)d.B * L * N);
        }
    }
    if (out) *out = w;
    return off;
}

// Bytes of workspace a handle of these dimensions allocates.
size_t workspace_need(const Dims& d) { return carve_work(d, nullptr, nullptr, true); }

struct Stage {
    double ms = 0;
    long long launches = 0;
};

}  // namespace

struct dv_handle {
    Dims d;
    int device = 0;
    int cus = 0;   // compute units of the device
    void* wmem = nullptr;   // weights
    void* ws = nullptr;     // workspace
    size_t ws_bytes = 0;
    // weights
    const void* W_pe;
    const float *b_pe, *cls, *pos, *lnf_g, *lnf_b;
    std::vector<LayerW> layers;
    Work w;                 // views into ws
    // stream state: frames seen since the last reset, their group size, and the cached
    // reference (stream frame index, -1 none); under reordering the number of held frames
    // (stream frames st_pos - st_hold .. st_pos - 1) and the mode and tau of the last call
    long long st_pos = 0;
    int st_G = 0;
    long long st_ref = -1;
    int st_hold = 0;
    int st_masks = -1;         // -1: no frame yet, 0: gate mode, 1: injected maps
    int st_mode = 0;
    float st_tau = 0.f;
    // profiling
    unsigned prof = 0;  // bit s: time stage s
    Stage stages[DV_NUM_STAGES];
    struct Pending {
        int stage;
        hipEvent_t a, b;
    };
    std::vector<Pending> pending;
    std::vector<hipEvent_t> pool;
};

namespace {

// ---- stage timing -----------------------------------------------------------------------------
struct Scope {
    dv_handle* h;
    int stage;
    hipStream_t s;
    hipEvent_t b = nullptr;
    Scope(dv_handle* h_, int st, hipStream_t s_) : h(h_), stage(st), s(s_) {
        if (!(h->prof >> stage & 1u)) return;
        hipEvent_t a = take(), bb = take();
        if (!a || !bb) return;
        (void)hipEventRecord(a, s);
        b = bb;
        h->pending.push_back({stage, a, bb});
    }
    ~Scope() {
        if (b) (void)hipEventRecord(b, s);
    }
    hipEvent_t take() {
        if (!h->pool.empty()) {
            hipEvent_t e = h->pool.back();
            h->pool.pop_back();
            return e;
        }
        hipEvent_t e = nullptr;
        if (hipEventCreate(&e) != hipSuccess) return nullptr;
        return e;
    }
};

int collect(dv_handle* h) {
    for (auto& p : h->pending) {
        HIP_TRY(hipEventSynchronize(p.b));
        float ms = 0.f;
        HIP_TRY(hipEventElapsedTime(&ms, p.a, p.b));
        h->stages[p.stage].ms += ms;
        h->stages[p.stage].launches += 1;
        h->pool.push_back(p.a);
        h->pool.push_back(p.b);
    }
    h->pending.clear();
    return DV_OK;
}

// ---- one batch of whole groups --------------------------------------------------------------
// frames, inj, emb, om, tokens start at local frame `skip`; frames below skip are carried over
// from an earlier call of a stream (local frame `cached`: the cached reference; the others stand
// for frames already returned).  fill >= 0: cache local frame fill, a reference needed by frames
// of the next call.  npend > 0: the first npend computed frames' pixels are at `pend`, the rest
// at `frames`.
int run_batch(dv_handle* h, Work& wk, const float* frames, int F, int G, int mode, float tau,
              const uint8_t* inj, float* emb, uint8_t* om, float* tokens, hipStream_t s,
              int skip = 0, int fill = -1, int cached = 0, const float* pend = nullptr,
              int npend = 0) {
    const Dims& d = h->d;
    const bool bf = d.bf16;
    const int N = d.N, D = d.D, L = d.L;
    const int T = F * N;
    const bool dense = mode == GATE_NONE;

    // identity row lists for the dense pass (built once per batch size)
    if (dense && wk.id_frames != F) {
        launch_compact(nullptr, nullptr, F, N, 1, wk.idx_id, wk.pos_id, wk.qoff_id, nullptr, s);
        wk.id_frames = F;
    }

    const size_t row_bytes = (size_t)N * D * sizeof(float);   // one frame's token rows
    const size_t el = bf ? 2 : 4;
    const size_t kv_bytes = (size_t)N * 2 * D * el;           // one frame's keys and values
    float* xs = wk.x + (size_t)skip * N * D;                  // the first computed frame's rows
    float* xcached = wk.x + (size_t)cached * N * D;
    if (skip > 0)   // the cached reference's layer-0 rows
        HIP_TRY(hipMemcpyAsync(xcached, wk.xc, row_bytes, hipMemcpyDeviceToDevice, s));
    {   // patch embedding + class-token rows
        Scope sc(h, DV_STAGE_PATCH, s);
        if (npend > 0)
            launch_im2col(bf, pend, npend, d.S, d.p, d.Kp, wk.A, s);
        if (F - skip > npend)
            launch_im2col(bf, frames, F - skip - npend, d.S, d.p, d.Kp,
                          (char*)wk.A + (size_t)npend * d.P * d.Kp * el, s);
        launch_cls_init(xs, h->cls, h->pos, F - skip, N, D, s);
        GemmArgs g{};
        g.A = wk.A;
        g.W = h->W_pe;
        g.bias = h->b_pe;
        g.K = d.Kp;
        g.Nout = D;
        g.Mdev = nullptr;
        g.Mconst = (F - skip) * d.P;
        g.Mmax = (F - skip) * d.P;
        g.cus = h->cus;
        g.out = xs;
        g.pos = h->pos;
        g.P = d.P;
        g.N = N;
        launch_gemm(Epi::Patch, bf, g, s);
    }

    const int* idx = dense ? wk.idx_id : wk.idx;
    const int* pos = dense ? wk.pos_id : wk.pos_;
    const int* qoff = dense ? wk.qoff_id : wk.qoff;
    const int* Mdev = dense ? nullptr : wk.M;
    // restoration of reused rows: on whenever tokens can be reused
    const bool restore = d.restore && !dense;
    // learned decision gate: gate mode only (injected maps and the sentinels bypass it)
    const bool decide = d.decision && mode == GATE_COS;
    const bool reord = d.reorder && !dense;
    // reordered without restoration: reused rows are aliases, resolved through the root map
    const bool alias = reord && !restore;

    for (int l = 0; l < L; ++l) {
        const LayerW& w = h->layers[l];
        uint8_t* cur = wk.mask[l & 1];
        uint8_t* prev = l > 0 ? wk.mask[(l - 1) & 1] : nullptr;
        if (fill >= 0)   // the layer input of a reference carried to the next call
            launch_copy_rows(wk.x, (alias && l > 0) ? wk.root : nullptr, fill, N, D,
                             wk.xc + (size_t)l * N * D, s);
        {   // reuse gate + LN1 of every recomputed token (reuse off: LN1 of every token)
            Scope sc(h, DV_STAGE_GATE, s);
            GateArgs ga{};
            ga.x = wk.x;
            ga.F = F;
            ga.N = N;
            ga.D = D;
            ga.G = G;
            ga.L = L;
            ga.layer = l;
            ga.mode = mode;
            ga.tau = tau;
            // restored rows differ from the reference's, and under reordering a token's source
            // may change from layer to layer: no shortcut from the previous map
            ga.prev = (mode == GATE_COS && !restore && !reord) ? prev : nullptr;
            ga.inj = inj;
            ga.cur = dense ? nullptr : cur;
            ga.out_masks = om;
            ga.cnt = dense ? nullptr : wk.cnt;
            ga.ln_g = w.ln1_g;
            ga.ln_b = w.ln1_b;
            ga.ln_out = wk.A;   // token-indexed LN1 rows; the QKV GEMM gathers them through idx
            ga.d_out = restore ? wk.A : nullptr;   // reused tokens' differences, same buffer
            ga.dec = decide ? w.dec : nullptr;
            ga.tcls = (decide && l > 0) ? wk.tcls : nullptr;
            ga.H = d.H;
            ga.reorder = reord;
            ga.src = reord ? wk.srcmap : nullptr;
            // restored rows are written out every layer; otherwise reused rows alias their root
            ga.root = (alias && l > 0) ? wk.root : nullptr;
            ga.skip = skip;
            launch_gate(bf, ga, s);
        }
        if (!dense) {
            Scope sc(h, DV_STAGE_COMPACT, s);
            launch_scan_compact(wk.cnt, gate_chunks(N), restore ? (F - skip) * N : 0, cur, F, N, G,
                                wk.idx, wk.pos_, wk.qoff, wk.M, restore ? wk.ridx : nullptr, s,
                                skip, wk.ext_row, restore && reord ? wk.rslot : nullptr);
            if (reord) launch_resolve(cur, wk.srcmap, F, N, G, wk.pos_, wk.root, s);
        }
        if (restore) {   // restoration hidden rows: GELU(dx W_r1^T + b_r1), before LN2 reuses A
            Scope sc(h, DV_STAGE_RESTORE, s);
            GemmArgs r{};
            r.A = wk.A;
            r.a_idx = wk.ridx;
            r.W = w.W_r1;
            r.bias = w.b_r1;
            r.K = D;
            r.Nout = RH;
            r.Mdev = wk.M + 1;
            r.Mconst = T;
            r.Mmax = T;
            r.cus = h->cus;
            r.out = wk.Hr;
            launch_gemm(Epi::Fc1, bf, r, s);
        }
        GemmArgs g{};
        g.Mdev = Mdev;
        g.Mconst = T;
        g.Mmax = T;
        g.cus = h->cus;
        g.idx = idx;
        {
            Scope sc(h, DV_STAGE_QKV, s);
            g.A = wk.A;
            g.a_idx = idx;   // packed row m is token row idx[m] of the LN1 buffer
            g.W = w.W_qkv;
            g.bias = w.b_qkv;
            g.K = D;
            g.Nout = 3 * D;
            g.out = wk.qkv;
            launch_gemm(Epi::Qkv, bf, g, s);
        }
        if (skip > 0)   // the cached reference's keys and values, at packed rows ext_row ..
            HIP_TRY(hipMemcpy2DAsync((char*)wk.qkv + ((size_t)wk.ext_row * 3 * D + D) * el,
                                     3 * D * el, (const char*)wk.kvc + (size_t)l * kv_bytes,
                                     2 * D * el, 2 * D * el, N, hipMemcpyDeviceToDevice, s));
        if (fill >= 0)
            launch_copy_ref_kv(wk.qkv, pos, fill, N, D, (int)el,
                               (char*)wk.kvc + (size_t)l * kv_bytes, s);
        g.a_idx = nullptr;
        AttnArgs at{};
        at.qkv = wk.qkv;
        at.pos = pos;
        at.qoff = qoff;
        at.out = wk.O;
        at.F = F;
        at.N = N;
        at.D = D;
        at.H = d.H;
        // per-group blocks assume the star with the reference's rows packed in the batch
        at.G = (dense || reord || skip > 0) ? 0 : G;
        at.skip = skip;
        at.sparse = !dense;
        at.cus = h->cus;
        {
            Scope sc(h, DV_STAGE_ATTN, s);
            launch_attention(bf, at, s);
        }
        if (decide && l + 1 < L) {   // the next layer's importance cue
            Scope sc(h, DV_STAGE_CLS, s);
            AttnArgs ac = at;
            ac.G = G;   // I frames are not gated
            launch_cls_attention(bf, ac, wk.tcls, s);
        }
        {
            Scope sc(h, DV_STAGE_OPROJ, s);
            g.A = wk.O;
            g.W = w.W_o;
            g.bias = w.b_o;
            g.K = D;
            g.Nout = D;
            g.out = wk.Z;
            g.resid = wk.x;
            launch_gemm(Epi::OProj, bf, g, s);
        }
        {
            Scope sc(h, DV_STAGE_LN2, s);
            launch_ln_rows(bf, wk.Z, nullptr, Mdev, T, D, w.ln2_g, w.ln2_b, wk.A, s);
        }
        {
            Scope sc(h, DV_STAGE_FC1, s);
            g.A = wk.A;
            g.W = w.W_1;
            g.bias = w.b_1;
            g.K = D;
            g.Nout = d.Dm;
            g.out = wk.Hb;
            g.resid = nullptr;
            launch_gemm(Epi::Fc1, bf, g, s);
        }
        {
            Scope sc(h, DV_STAGE_FC2, s);
            g.A = wk.Hb;
            g.W = w.W_2;
            g.bias = w.b_2;
            g.K = d.Dm;
            g.Nout = D;
            g.out = wk.x;
            g.resid = wk.Z;
            launch_gemm(Epi::Fc2, bf, g, s);
        }
        if (skip > 0)   // the cached reference's new rows, for the restoration, merges, next gate
            HIP_TRY(hipMemcpyAsync(xcached, wk.xc + (size_t)(l + 1) * N * D, row_bytes,
                                   hipMemcpyDeviceToDevice, s));
        if (restore && reord) {   // restoration outputs, then each reused row along its chain
            Scope sc(h, DV_STAGE_RESTORE, s);
            GemmArgs r{};
            r.A = wk.Hr;
            r.W = w.W_r2;
            r.bias = w.b_r2;
            r.K = RH;
            r.Nout = D;
            r.Mdev = wk.M + 1;
            r.Mconst = T;
            r.Mmax = T;
            r.cus = h->cus;
            r.out = wk.rbuf;
            launch_gemm(Epi::Delta, bf, r, s);
            launch_restore_chain(wk.x, wk.rbuf, wk.ridx, wk.rslot, cur, wk.srcmap, wk.M + 1, T, F,
                                 N, D, G, s);
        } else if (restore) {   // reused rows: the reference token's new row + Hr W_r2^T + b_r2
            Scope sc(h, DV_STAGE_RESTORE, s);
            GemmArgs r{};
            r.A = wk.Hr;
            r.W = w.W_r2;
            r.bias = w.b_r2;
            r.K = RH;
            r.Nout = D;
            r.Mdev = wk.M + 1;
            r.Mconst = T;
            r.Mmax = T;
            r.cus = h->cus;
            r.idx = wk.ridx;
            r.resid = wk.x;
            r.out = wk.x;
            r.N = N;
            r.G = G;
            launch_gemm(Epi::Restore, bf, r, s);
        } else if (reord) {
            // reused rows stay aliases of the frame that recomputed them (the root map); they
            // are filled in only to hand out the tokens
            if (tokens && l == L - 1) {
                Scope sc(h, DV_STAGE_MERGE, s);
                launch_merge(wk.x, cur, wk.root, F, N, D, G, s);
            }
        } else if (mode == GATE_INJECT || mode == GATE_ALL ||
                   (mode == GATE_COS && tokens && l == L - 1)) {
            // reused rows take the reference's new row (gate mode: only to hand out tokens)
            Scope sc(h, DV_STAGE_MERGE, s);
            launch_merge(wk.x, cur, nullptr, F, N, D, G, s);
        }
        if (fill >= 0 && l == L - 1)   // the reference's last-layer rows (restored ones included)
            launch_copy_rows(wk.x, alias ? wk.root : nullptr, fill, N, D,
                             wk.xc + (size_t)L * N * D, s);
    }
    {
        Scope sc(h, DV_STAGE_FINAL, s);
        launch_final_ln(xs, F - skip, N, D, h->lnf_g, h->lnf_b, emb, s);
    }
    if (tokens)
        HIP_TRY(hipMemcpyAsync(tokens, xs, (size_t)(F - skip) * row_bytes, hipMemcpyDeviceToDevice,
                               s));
    return DV_OK;
}

// Validates the arguments of an encode call; sets *mode.
int check_encode(const dv_handle* h, const float* frames, int n, int G, float tau,
                 const uint8_t* masks, const float* emb, int* mode) {
    if (!h) return fail(DV_EINVAL, "handle is NULL");
    if (!frames || !emb) return fail(DV_EINVAL, "frames and out_embeddings must not be NULL");
    if (n < 1) return fail(DV_EINVAL, "n_frames must be >= 1 (got %d)", n);
    if (G < 1) return fail(DV_EINVAL, "group_size must be >= 1 (got %d)", G);
    if (G > h->d.B) return fail(DV_EINVAL, "group_size %d exceeds max_batch_frames %d", G, h->d.B);
    if (masks) {
        *mode = GATE_INJECT;
    } else {
        if (std::isnan(tau)) return fail(DV_EINVAL, "tau is NaN");
        *mode = (tau == -INFINITY) ? GATE_NONE : (tau == INFINITY) ? GATE_ALL : GATE_COS;
    }
    const Dims& d = h->d;
    if (d.reorder && G % 4)
        return fail(DV_EINVAL, "reordered referencing needs a group_size that is a multiple of 4 "
                    "(got %d)", G);
    if (d.reorder && d.restore && G / 4 + 1 > CHAIN_MAX)
        return fail(DV_EINVAL, "reordered referencing with restoration supports group_size <= %d "
                    "(got %d)", 4 * (CHAIN_MAX - 1), G);
    return DV_OK;
}

// An encode call over internal batches of at most `batch` frames (whole groups) with workspace
// w, laid out for that many frames.  Arguments already checked.
int encode_batches(dv_handle* h, Work& w, int batch, const float* frames, int n, int G, int mode,
                   float tau, const uint8_t* masks, float* emb, uint8_t* om, float* tokens,
                   hipStream_t s) {
    const Dims& d = h->d;
    const int per = (batch / G) * G;
    const size_t img = (size_t)3 * d.S * d.S;
    HIP_TRY(hipSetDevice(h->device));
    for (int f0 = 0; f0 < n; f0 += per) {
        const int F0 = std::min(per, n - f0);
        // reordering: the next batch's first frame, an I frame, closes this batch's last block
        // (its results are computed again, identically, as part of the next batch)
        const int F = F0 + (d.reorder && f0 + F0 < n ? 1 : 0);
        const size_t ml = (size_t)d.L * d.N;
        int rc = run_batch(h, w, frames + (size_t)f0 * img, F, G, mode, tau,
                           masks ? masks + (size_t)f0 * ml : nullptr, emb + (size_t)f0 * d.D,
                           om ? om + (size_t)f0 * ml : nullptr,
                           tokens ? tokens + (size_t)f0 * d.N * d.D : nullptr, s);
        if (rc) return rc;
    }
    HIP_TRY(hipGetLastError());
    return DV_OK;
}

// An encode call with the handle's own workspace.
int encode_impl(dv_handle* h, const float* frames, int n, int G, float tau, const uint8_t* masks,
                float* emb, uint8_t* om, float* tokens, hipStream_t s) {
    int mode;
    int rc = check_encode(h, frames, n, G, tau, masks, emb, &mode);
    if (rc) return rc;
    return encode_batches(h, h->w, h->d.B, frames, n, G, mode, tau, masks, emb, om, tokens, s);
}

// A reordered stream.  A frame between anchors a and a + 4 (stream indices that are multiples of
// 4) references the later one, so the frames after the last anchor received are held (at most 3)
// and encoded by the call that brings their anchor, or by a flush, which encodes them as the
// stream's last frames (no later anchor) and ends the stream.  A call outputs the frames it
// completes, in stream order: the held ones, then its own up to its last anchor.  Each batch
// starts at a group boundary: the frames before the first one computed are carried over (the
// last of them, the anchor of the first computed frame, from the cache), and ends on an anchor,
// which is cached for the next batch.
int stream_reorder_impl(dv_handle* h, const float* frames, int n, int G, int mode, float tau,
                        const uint8_t* masks, float* emb, uint8_t* om, float* tokens,
                        hipStream_t s, bool flush) {
    const Dims& d = h->d;
    if (d.B <= G)
        return fail(DV_EINVAL, "streaming with reordered referencing needs max_batch_frames > "
                    "group_size (%d <= %d)", d.B, G);
    const size_t img = (size_t)3 * d.S * d.S, ml = (size_t)d.L * d.N, N = d.N, D = d.D;
    const long long st = h->st_pos;                   // frames received before this call
    const long long total = st + n;
    const long long done = st - h->st_hold;           // the first frame not yet output
    const long long last = flush ? total - 1 : (total - 1) / 4 * 4;   // the last it completes
    for (long long u = done; u <= last;) {
        int lead = 0;   // carried-over frames: the gaps since the group start, then the anchor
        if (u % G != 0 && mode != GATE_NONE) {
            if (h->st_ref != u - 1)
                return fail(DV_EINVAL, "the stream lost its cached reference (an earlier call "
                            "failed?): call dv_stream_reset");
            lead = (int)(u - (u - 1) / G * G);
        }
        long long cnt = std::min<long long>(d.B - lead, last - u + 1);
        if (u + cnt - 1 < last) cnt = (u + cnt - 1) / 4 * 4 - u + 1;   // end on an anchor
        if (cnt < 1) return fail(DV_EINVAL, "internal: empty stream batch");
        const long long e = u + cnt - 1;
        const int F = lead + (int)cnt;
        const int npend = (int)std::max<long long>(0, std::min(st, e + 1) - u);
        const float* pend = npend ? h->w.hold + (size_t)(u - done) * img : nullptr;
        const float* fr = frames ? frames + (size_t)std::max<long long>(0, u - st) * img : nullptr;
        const uint8_t* inj = nullptr;
        if (masks || (flush && mode == GATE_INJECT)) {
            if (npend) {   // held frames' maps, then the call's own
                HIP_TRY(hipMemcpyAsync(h->w.injs, h->w.holdm + (size_t)(u - done) * ml, npend * ml,
                                       hipMemcpyDeviceToDevice, s));
                if (cnt > npend)
                    HIP_TRY(hipMemcpyAsync(h->w.injs + npend * ml, masks, (cnt - npend) * ml,
                                           hipMemcpyDeviceToDevice, s));
                inj = h->w.injs;
            } else {
                inj = masks + (size_t)(u - st) * ml;
            }
        }
        const size_t k = (size_t)(u - done);
        const int fill = flush ? -1 : F - 1;
        int rc = run_batch(h, h->w, fr, F, G, mode, tau, inj, emb + k * D,
                           om ? om + k * ml : nullptr,
                           tokens ? tokens + k * N * D : nullptr, s, lead, fill,
                           lead > 0 ? lead - 1 : 0, pend, npend);
        if (rc) return rc;
        if (fill >= 0) h->st_ref = e;
        u = e + 1;
    }
    if (flush) {
        h->st_pos = 0;
        h->st_hold = 0;
        h->st_ref = -1;
        h->st_masks = -1;
        return DV_OK;
    }
    // the frames after the last anchor wait for the next call; those held already stay in place
    // (when this call completed nothing) or are all replaced by frames of this call
    const long long h0 = last + 1;
    for (long long g = std::max(h0, st); g < total; ++g) {
        HIP_TRY(hipMemcpyAsync(h->w.hold + (size_t)(g - h0) * img, frames + (size_t)(g - st) * img,
                               img * sizeof(float), hipMemcpyDeviceToDevice, s));
        if (masks)
            HIP_TRY(hipMemcpyAsync(h->w.holdm + (size_t)(g - h0) * ml, masks + (size_t)(g - st) * ml,
                                   ml, hipMemcpyDeviceToDevice, s));
    }
    h->st_hold = (int)(total - h0);
    h->st_pos = total;
    h->st_G = G;
    h->st_masks = masks ? 1 : 0;
    h->st_mode = mode;
    h->st_tau = tau;
    return DV_OK;
}

// A stream call: frames get stream indices st_pos .. st_pos + n - 1; frame g's reference is
// frame G * floor(g / G), possibly from an earlier call (then read from the cache).
int stream_impl(dv_handle* h, const float* frames, int n, int G, float tau, const uint8_t* masks,
                float* emb, uint8_t* om, float* tokens, hipStream_t s) {
    if (!h) return fail(DV_EINVAL, "handle is NULL");
    if (!frames || !emb) return fail(DV_EINVAL, "frames and out_embeddings must not be NULL");
    if (n < 1) return fail(DV_EINVAL, "n_frames must be >= 1 (got %d)", n);
    if (G < 1) return fail(DV_EINVAL, "group_size must be >= 1 (got %d)", G);
    const Dims& d = h->d;
    if (G > d.B) return fail(DV_EINVAL, "group_size %d exceeds max_batch_frames %d", G, d.B);
    if (h->st_pos > 0 && G != h->st_G)
        return fail(DV_EINVAL, "group_size %d differs from the stream's %d (dv_stream_reset "
                    "starts a new stream)", G, h->st_G);
    int mode;
    if (masks) {
        mode = GATE_INJECT;
    } else {
        if (std::isnan(tau)) return fail(DV_EINVAL, "tau is NaN");
        mode = (tau == -INFINITY) ? GATE_NONE : (tau == INFINITY) ? GATE_ALL : GATE_COS;
    }
    if (d.reorder && G % 4)
        return fail(DV_EINVAL, "reordered referencing needs a group_size that is a multiple of 4 "
                    "(got %d)", G);
    if (d.reorder && d.restore && G / 4 + 1 > CHAIN_MAX)
        return fail(DV_EINVAL, "reordered referencing with restoration supports group_size <= %d "
                    "(got %d)", 4 * (CHAIN_MAX - 1), G);
    if (d.reorder && h->st_hold > 0 && (masks != nullptr) != (h->st_masks == 1))
        return fail(DV_EINVAL, "a reordered stream holding frames cannot switch between gate "
                    "mode and injected maps");
    HIP_TRY(hipSetDevice(h->device));
    if (d.reorder) {
        int rc = stream_reorder_impl(h, frames, n, G, mode, tau, masks, emb, om, tokens, s, false);
        if (rc) return rc;
        HIP_TRY(hipGetLastError());
        return DV_OK;
    }
    const size_t N = d.N, D = d.D, L = d.L;
    const size_t img = (size_t)3 * d.S * d.S, ml = L * N;
    const long long g0 = h->st_pos;
    const long long last = (g0 + n - 1) / G * G;   // the last group's reference
    const bool open = g0 + n < last + G;           // ... whose group continues after this call
    for (int k = 0; k < n;) {
        const long long gk = g0 + k, gs = gk / G * G;
        int lead = 0;   // carried-over frames ahead of frame gk: its reference and the gaps
        if (gs < gk && mode != GATE_NONE) {
            if (h->st_ref != gs)
                return fail(DV_EINVAL, "the stream lost its cached reference (an earlier call "
                            "failed?): call dv_stream_reset");
            lead = (int)(gk - gs);
        }
        int cnt = std::min(d.B - lead, n - k);
        if (k + cnt < n) cnt = (int)((gk + cnt) / G * G - gk);   // end on a group boundary
        const int fill = (open && last >= gk && last < gk + cnt) ? (int)(last - gk) + lead : -1;
        int rc = run_batch(h, h->w, frames + (size_t)k * img, lead + cnt, G, mode, tau,
                           masks ? masks + (size_t)k * ml : nullptr, emb + (size_t)k * D,
                           om ? om + (size_t)k * ml : nullptr,
                           tokens ? tokens + (size_t)k * N * D : nullptr, s, lead, fill);
        if (rc) return rc;
        if (fill >= 0) h->st_ref = last;
        k += cnt;
    }
    h->st_pos = g0 + n;
    h->st_G = G;
    HIP_TRY(hipGetLastError());
    return DV_OK;
}

template <class T>
T* carve(char*& p, size_t count) {
    T* r = (T*)p;
    p += round_up(count * sizeof(T), 256);
    return r;
}

}  // namespace

extern "C" {

size_t dv_weights_floats(const dv_config* cfg) {
    Dims d;
    std::string keep = g_err;
    if (check_config(cfg, &d) != DV_OK) {
        g_err = keep;
        return 0;
    }
    return blob_floats(d);
}

const char* dv_last_error(void) { return g_err.c_str(); }

int dv_create(const dv_config* cfg, const float* weights, size_t weights_bytes, dv_handle** out) {
    if (!out) return fail(DV_EINVAL, "out is NULL");
    *out = nullptr;
    Dims d;
    int rc = check_config(cfg, &d);
    if (rc) return rc;
    if (!weights) return fail(DV_EINVAL, "weights is NULL");
    const size_t nf = blob_floats(d);
    if (weights_bytes != nf * sizeof(float))
        return fail(DV_EINVAL, "weight blob has %zu bytes, configuration needs %zu", weights_bytes,
                    nf * sizeof(float));
    const bool bf = d.bf16;
    const size_t el = bf ? 2 : 4;
    const size_t D = d.D, Dm = d.Dm, N = d.N, L = d.L;

    // --- weights: matrices in elem (bf16 rounded or fp32), vectors in fp32 -------------------
    std::vector<char> host;
    struct Off { size_t o; };
    size_t wbytes = 0;
    auto reserve = [&](size_t bytes) {
        size_t o = wbytes;
        wbytes += round_up(bytes, 256);
        return o;
    };
    const size_t o_pe = reserve(D * d.Kp * el), o_bpe = reserve(D * 4), o_cls = reserve(D * 4),
                 o_pos = reserve(N * D * 4);
    struct LO { size_t ln1_g, ln1_b, W_qkv, b_qkv, W_o, b_o, ln2_g, ln2_b, W_1, b_1, W_2, b_2; };
    std::vector<LO> lo(L);
    for (size_t l = 0; l < L; ++l) {
        lo[l].ln1_g = reserve(D * 4);
        lo[l].ln1_b = reserve(D * 4);
        lo[l].W_qkv = reserve(3 * D * D * el);
        lo[l].b_qkv = reserve(3 * D * 4);
        lo[l].W_o = reserve(D * D * el);
        lo[l].b_o = reserve(D * 4);
        lo[l].ln2_g = reserve(D * 4);
        lo[l].ln2_b = reserve(D * 4);
        lo[l].W_1 = reserve(Dm * D * el);
        lo[l].b_1 = reserve(Dm * 4);
        lo[l].W_2 = reserve(D * Dm * el);
        lo[l].b_2 = reserve(D * 4);
    }
    const size_t o_lnf_g = reserve(D * 4), o_lnf_b = reserve(D * 4);
    struct RO { size_t W_r1, b_r1, W_r2, b_r2; };
    std::vector<RO> ro(d.restore ? L : 0);
    for (auto& r : ro) {
        r.W_r1 = reserve(RH * D * el);
        r.b_r1 = reserve(RH * 4);
        r.W_r2 = reserve(D * RH * el);
        r.b_r2 = reserve(D * 4);
    }
    std::vector<size_t> dco(d.decision ? L : 0);
    for (auto& o : dco) o = reserve(DEC_FLOATS * 4);
    // an optional cap on the device memory a handle may take (weights and workspace), checked
    // before any device call: DV_MAX_DEVICE_BYTES in the environment
    if (const char* cap = getenv("DV_MAX_DEVICE_BYTES")) {
        const unsigned long long c = strtoull(cap, nullptr, 10);
        if (wbytes + workspace_need(d) > c)
            return fail(DV_ENOMEM, "the handle needs %zu bytes of device memory, above "
                        "DV_MAX_DEVICE_BYTES=%llu", wbytes + workspace_need(d), c);
    }
    try {
        host.assign(wbytes, 0);
    } catch (const std::bad_alloc&) {
        return fail(DV_ENOMEM, "host staging buffer of %zu bytes", wbytes);
    }
    const float* src = weights;
    auto put_vec = [&](size_t off, size_t count) {
        memcpy(host.data() + off, src, count * 4);
        src += count;
    };
    auto put_mat = [&](size_t off, size_t rows, size_t cols, size_t ld) {
        for (size_t r = 0; r < rows; ++r)
            for (size_t c = 0; c < cols; ++c) {
                const float v = src[r * cols + c];
                if (bf) ((uint16_t*)(host.data() + off))[r * ld + c] = f32_to_bf16(v);
                else ((float*)(host.data() + off))[r * ld + c] = v;
            }
        src += rows * cols;
    };
    put_mat(o_pe, D, 3 * (size_t)d.p * d.p, d.Kp);  // [D, 3p^2] padded to Kp with zeros
    put_vec(o_bpe, D);
    put_vec(o_cls, D);
    put_vec(o_pos, N * D);
    for (size_t l = 0; l < L; ++l) {
        put_vec(lo[l].ln1_g, D);
        put_vec(lo[l].ln1_b, D);
        put_mat(lo[l].W_qkv, 3 * D, D, D);
        put_vec(lo[l].b_qkv, 3 * D);
        put_mat(lo[l].W_o, D, D, D);
        put_vec(lo[l].b_o, D);
        put_vec(lo[l].ln2_g, D);
        put_vec(lo[l].ln2_b, D);
        put_mat(lo[l].W_1, Dm, D, D);
        put_vec(lo[l].b_1, Dm);
        put_mat(lo[l].W_2, D, Dm, Dm);
        put_vec(lo[l].b_2, D);
    }
    put_vec(o_lnf_g, D);
    put_vec(o_lnf_b, D);
    for (auto& r : ro) {
        put_mat(r.W_r1, RH, D, D);
        put_vec(r.b_r1, RH);
        put_mat(r.W_r2, D, RH, RH);
        put_vec(r.b_r2, D);
    }
    for (auto o : dco) put_vec(o, DEC_FLOATS);   // W_d1, b_d1, W_d2, b_d2 as the kernel reads them

    dv_handle* h = new (std::nothrow) dv_handle();
    if (!h) return fail(DV_ENOMEM, "handle");
    h->d = d;
    auto cleanup = [&](int code) {
        if (h->wmem) (void)hipFree(h->wmem);
        if (h->ws) (void)hipFree(h->ws);
        delete h;
        return code;
    };
    if (hipGetDevice(&h->device) != hipSuccess) return cleanup(fail(DV_EHIP, "hipGetDevice failed"));
    scratch_setup(h->device);   // dv_encode_noalloc's array on this device (errors reported there)
    if (hipDeviceGetAttribute(&h->cus, hipDeviceAttributeMultiprocessorCount, h->device) !=
        hipSuccess)
        h->cus = 0;   // the GEMMs then keep one tiling for all rows
    {
        hipError_t e = hipMalloc(&h->wmem, wbytes);
        if (e != hipSuccess) {
            h->wmem = nullptr;
            return cleanup(fail(e == hipErrorOutOfMemory ? DV_ENOMEM : DV_EHIP, "weights: %s",
                                hipGetErrorString(e)));
        }
        e = hipMemcpy(h->wmem, host.data(), wbytes, hipMemcpyHostToDevice);
        if (e != hipSuccess) return cleanup(fail(DV_EHIP, "weight upload: %s", hipGetErrorString(e)));
    }
    char* wb = (char*)h->wmem;
    h->W_pe = wb + o_pe;
    h->b_pe = (const float*)(wb + o_bpe);
    h->cls = (const float*)(wb + o_cls);
    h->pos = (const float*)(wb + o_pos);
    h->lnf_g = (const float*)(wb + o_lnf_g);
    h->lnf_b = (const float*)(wb + o_lnf_b);
    h->layers.resize(L);
    for (size_t l = 0; l < L; ++l) {
        LayerW& w = h->layers[l];
        w.ln1_g = (const float*)(wb + lo[l].ln1_g);
        w.ln1_b = (const float*)(wb + lo[l].ln1_b);
        w.W_qkv = wb + lo[l].W_qkv;
        w.b_qkv = (const float*)(wb + lo[l].b_qkv);
        w.W_o = wb + lo[l].W_o;
        w.b_o = (const float*)(wb + lo[l].b_o);
        w.ln2_g = (const float*)(wb + lo[l].ln2_g);
        w.ln2_b = (const float*)(wb + lo[l].ln2_b);
        w.W_1 = wb + lo[l].W_1;
        w.b_1 = (const float*)(wb + lo[l].b_1);
        w.W_2 = wb + lo[l].W_2;
        w.b_2 = (const float*)(wb + lo[l].b_2);
        w.W_r1 = w.W_r2 = nullptr;
        w.b_r1 = w.b_r2 = nullptr;
        if (d.restore) {
            w.W_r1 = wb + ro[l].W_r1;
            w.b_r1 = (const float*)(wb + ro[l].b_r1);
            w.W_r2 = wb + ro[l].W_r2;
            w.b_r2 = (const float*)(wb + ro[l].b_r2);
        }
        w.dec = d.decision ? (const float*)(wb + dco[l]) : nullptr;
    }

    // --- workspace (with the stream state, so that no encode call allocates) -----------------
    const size_t need = workspace_need(d);
    {
        hipError_t e = hipMalloc(&h->ws, need);
        if (e != hipSuccess) {
            h->ws = nullptr;
            return cleanup(fail(e == hipErrorOutOfMemory ? DV_ENOMEM : DV_EHIP,
                                "workspace of %zu bytes: %s", need, hipGetErrorString(e)));
        }
        // defined contents in the row padding that GEMM tiles read past M
        e = hipMemset(h->ws, 0, need);
        if (e != hipSuccess) return cleanup(fail(DV_EHIP, "workspace clear: %s", hipGetErrorString(e)));
    }
    h->ws_bytes = need;
    carve_work(d, (char*)h->ws, &h->w, true);
    *out = h;
    return DV_OK;
}

int dv_destroy(dv_handle* h) {
    if (!h) return DV_OK;
    (void)hipSetDevice(h->device);
    (void)hipDeviceSynchronize();
    for (auto& pe : h->pending) {
        (void)hipEventDestroy(pe.a);
        (void)hipEventDestroy(pe.b);
    }
    for (auto e : h->pool) (void)hipEventDestroy(e);
    if (h->wmem) (void)hipFree(h->wmem);
    if (h->ws) (void)hipFree(h->ws);
    delete h;
    return DV_OK;
}

int dv_workspace_bytes(const dv_handle* h, size_t* bytes) {
    if (!h || !bytes) return fail(DV_EINVAL, "NULL argument");
    *bytes = h->ws_bytes;
    return DV_OK;
}

int dv_encode(dv_handle* h, const float* frames, int n_frames, int group_size, float tau,
              float* out_embeddings, uint8_t* out_masks, hipStream_t stream) {
    return encode_impl(h, frames, n_frames, group_size, tau, nullptr, out_embeddings, out_masks,
                       nullptr, stream);
}

int dv_encode_noalloc(dv_handle* h, const float* frames, int n_frames, int group_size, float tau,
                      float* out_embeddings, uint8_t* out_masks, hipStream_t stream) {
    int mode;
    int rc = check_encode(h, frames, n_frames, group_size, tau, nullptr, out_embeddings, &mode);
    if (rc) return rc;
    void* base = scratch_base(h->device);
    if (!base)
        return fail(DV_EHIP, "the scratch array of device %d has no address (set-up failed: %s)",
                    h->device, g_scratch_err.c_str());
    // internal batches: as many whole groups as the scratch holds, at most max_batch_frames
    Dims dn = h->d;
    int best = 0;
    for (int b = group_size; b <= h->d.B; b += group_size) {
        dn.B = b;
        dn.Bw = b + (dn.reorder ? 1 : 0);
        if (carve_work(dn, nullptr, nullptr, false) > DV_SCRATCH_BYTES) break;
        best = b;
    }
    if (best == 0) {
        dn.B = group_size;
        dn.Bw = group_size + (dn.reorder ? 1 : 0);
        return fail(DV_ENOMEM, "one group of %d frames needs %zu bytes of scratch, above the %llu "
                    "bytes of dv_encode_noalloc's static array", group_size,
                    carve_work(dn, nullptr, nullptr, false), (unsigned long long)DV_SCRATCH_BYTES);
    }
    dn.B = best;
    dn.Bw = best + (dn.reorder ? 1 : 0);
    Work w;
    carve_work(dn, (char*)base, &w, false);   // identity lists are rebuilt: another call may
    w.id_frames = -1;                        // have used the array since
    const unsigned prof = h->prof;            // stage timing creates events: off for this call
    h->prof = 0;
    rc = encode_batches(h, w, best, frames, n_frames, group_size, mode, tau, nullptr,
                        out_embeddings, out_masks, nullptr, stream);
    h->prof = prof;
    return rc;
}

int dv_encode_masked(dv_handle* h, const float* frames, int n_frames, int group_size,
                     const uint8_t* masks, float* out_embeddings, uint8_t* out_masks,
                     hipStream_t stream) {
    if (!masks) return fail(DV_EINVAL, "masks is NULL");
    return encode_impl(h, frames, n_frames, group_size, 0.f, masks, out_embeddings, out_masks,
                       nullptr, stream);
}

int dv_encode_tokens(dv_handle* h, const float* frames, int n_frames, int group_size, float tau,
                     const uint8_t* masks, float* out_embeddings, uint8_t* out_masks,
                     float* out_tokens, hipStream_t stream) {
    return encode_impl(h, frames, n_frames, group_size, tau, masks, out_embeddings, out_masks,
                       out_tokens, stream);
}

int dv_stream_encode(dv_handle* h, const float* frames, int n_frames, int group_size, float tau,
                     const uint8_t* masks, float* out_embeddings, uint8_t* out_masks,
                     float* out_tokens, hipStream_t stream) {
    return stream_impl(h, frames, n_frames, group_size, tau, masks, out_embeddings, out_masks,
                       out_tokens, stream);
}

int dv_stream_reset(dv_handle* h) {
    if (!h) return fail(DV_EINVAL, "handle is NULL");
    h->st_pos = 0;
    h->st_G = 0;
    h->st_ref = -1;
    h->st_hold = 0;
    h->st_masks = -1;
    return DV_OK;
}

int dv_stream_held(const dv_handle* h, int* n_held) {
    if (!h || !n_held) return fail(DV_EINVAL, "handle and n_held must not be NULL");
    *n_held = h->st_hold;
    return DV_OK;
}

int dv_stream_flush(dv_handle* h, float* out_embeddings, uint8_t* out_masks, float* out_tokens,
                    hipStream_t stream) {
    if (!h) return fail(DV_EINVAL, "handle is NULL");
    if (h->st_hold > 0 && !out_embeddings)
        return fail(DV_EINVAL, "out_embeddings must not be NULL while frames are held");
    if (h->st_hold > 0) {
        HIP_TRY(hipSetDevice(h->device));
        int rc = stream_reorder_impl(h, nullptr, 0, h->st_G, h->st_mode, h->st_tau, nullptr,
                                     out_embeddings, out_masks, out_tokens, stream, true);
        if (rc) return rc;
        HIP_TRY(hipGetLastError());
    }
    return dv_stream_reset(h);
}

int dv_compact(const uint8_t* masks, int n_frames, int n_tokens, int group_size, int32_t* idx,
               int32_t* pos, int32_t* qoff, int32_t* count, hipStream_t stream) {
    if (!masks || !idx || !pos || !qoff || !count) return fail(DV_EINVAL, "NULL argument");
    if (n_frames < 1 || n_tokens < 1 || group_size < 1) return fail(DV_EINVAL, "sizes must be >= 1");
    if ((long long)n_frames * n_tokens > (1ll << 30)) return fail(DV_EINVAL, "too many tokens");
    // per-frame counts land in qoff[0..n) and are turned into the prefix in place by one block
    launch_count(masks, n_frames, n_tokens, group_size, qoff, stream);
    launch_scan(qoff, 1, n_frames, 0, qoff, count, stream);
    launch_compact(masks, qoff, n_frames, n_tokens, group_size, idx, pos, nullptr, nullptr,
                   stream);
    HIP_TRY(hipGetLastError());
    return DV_OK;
}

int dv_mfma_probe(int blocks, int iters, float* sink, double* flops, hipStream_t stream) {
    if (!sink || !flops) return fail(DV_EINVAL, "NULL argument");
    if (blocks < 1 || iters < 1 || blocks > (1 << 20)) return fail(DV_EINVAL, "blocks in [1, 2^20], iters >= 1");
    *flops = launch_mfma_loop(blocks, iters, sink, stream);
    HIP_TRY(hipGetLastError());
    return DV_OK;
}

int dv_profile(dv_handle* h, unsigned stage_mask) {
    if (!h) return fail(DV_EINVAL, "handle is NULL");
    int rc = collect(h);
    if (rc) return rc;
    for (auto& st : h->stages) st = Stage();
    h->prof = stage_mask & DV_PROFILE_ALL;
    return DV_OK;
}

int dv_profile_read(dv_handle* h, int stage, double* total_ms, long long* launches) {
    if (!h || !total_ms || !launches) return fail(DV_EINVAL, "NULL argument");
    if (stage < 0 || stage >= DV_NUM_STAGES) return fail(DV_EINVAL, "stage %d out of range", stage);
    int rc = collect(h);
    if (rc) return rc;
    *total_ms = h->stages[stage].ms;
    *launches = h->stages[stage].launches;
    return DV_OK;
}

}  // extern "C"
