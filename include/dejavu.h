/*
 * dejavu.h -- C ABI of the reuse-aware ViT encoder for AMD Instinct MI355X (gfx950).
 *
 * The library computes the ViT embedding of every frame of a video batch while
 * reusing per-token work across frames, following "DejaVu: Efficient
 * Video-Language Query Engine with Learning-based Inter-Frame Computation
 * Reuse" (PVLDB 18(10), 2025):
 *
 *   - ViT backbone: patch embedding, class token, learned position table, L
 *     pre-norm encoder layers, final LayerNorm of the class token
 *     (Section 2.3, ViT architecture figure).
 *   - Frames are cut into groups of G consecutive frames; the first frame of
 *     a group is the reference and is computed in full at every layer (the
 *     periodic full recompute of Section 6.3; a star form of the reference
 *     structure of Section 3.1).
 *   - Per layer and token, a reuse decision (Section 3.3, similarity cue of
 *     Eq. 1 with one reference and the hard gate M_i = [d_i > 0]) with the
 *     learned decision MLP replaced by a threshold: token i of a
 *     non-reference frame is reused when cos(x_f[i], x_ref[i]) >= tau, on the
 *     layer input x (residual stream) -- or, with DV_FLAG_DECISION, by the
 *     decision MLP itself.  The class token is never reused.
 *   - Token filtration (Section 3.3): recompute tokens are stream-compacted
 *     across all frames of the batch into dense rows (sparse computation
 *     compaction, Section 5.3) and run the whole encoder layer (QKV
 *     projection, attention over all N keys/values of the frame -- fresh rows
 *     for recomputed tokens, the reference's rows for reused ones --, output
 *     projection, MLP) on those rows only.
 *   - Token reconstruction (Section 3.3): reused tokens take the reference's
 *     layer output -- with DV_FLAG_RESTORE calibrated by the restoration
 *     layer (Section 3.3): plus a two-layer MLP (hidden 128, GELU) of the
 *     difference between the token's layer input and the reference's; reused
 *     keys and values stay the reference's.  Layers run over the whole batch one at a time
 *     (layer-wise scheduling, Section 5.1); the reference's per-layer state
 *     lives in the batch buffers for one layer step only (cached memory
 *     compaction, Section 5.2).
 *
 * Cosine convention: a.b / max(|a||b|, 1e-8) in fp32, clamped to [-1, 1],
 * and exactly 1 when the two rows are elementwise equal.
 *
 * Conventions for every entry point:
 *   - Return value: DV_OK (0) or a negative DV_E* code; dv_last_error() gives
 *     a message for the calling thread.
 *   - Arguments are validated on the host before any work is enqueued; on a
 *     validation error nothing is launched and no device memory is touched.
 *   - "device" pointers are HIP device allocations on the current device;
 *     "host" pointers are ordinary host memory.  The caller owns every buffer
 *     it passes; outputs must not alias inputs.
 *   - All layouts are dense, row-major, little-endian.
 *   - A handle is not re-entrant: use one handle per concurrently used stream.
 */
#ifndef DEJAVU_H
#define DEJAVU_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
#define DV_OK 0
#define DV_EINVAL (-1)        /* bad argument: null pointer, size < 1, NaN tau, size mismatch */
#define DV_ENOMEM (-2)        /* a device or host allocation failed */
#define DV_EHIP (-3)          /* a HIP runtime call failed (message names it) */
#define DV_EUNSUPPORTED (-4)  /* configuration outside what the kernels support */

/* arithmetic type of the GEMM and attention operands (the residual stream,
 * LayerNorm statistics, softmax and the reuse gate are always fp32) */
#define DV_F32 0
#define DV_BF16 1

typedef struct dv_config {
    int image_size;        /* S: frames are 3 x S x S */
    int patch;             /* p: S % p == 0; P = (S/p)^2 patches, N = P + 1 tokens */
    int depth;             /* L encoder layers */
    int width;             /* D */
    int heads;             /* H: D % H == 0, head dim D/H a multiple of 16 and <= 128 */
    int mlp;               /* Dm: MLP hidden width */
    int dtype;             /* DV_F32 or DV_BF16 */
    int max_batch_frames;  /* frames per internal batch (rounded down to whole groups per call) */
    unsigned flags;        /* DV_FLAG_RESTORE, DV_FLAG_DECISION, DV_FLAG_REORDER or 0 */
} dv_config;

/* Restoration layer on reused tokens (Section 3.3): after each layer, a reused token i of a
 * non-reference frame f becomes  y_ref[i] + W_r2 GELU(W_r1 (x_f[i] - x_ref[i]) + b_r1) + b_r2,
 * where x is the layer input and y_ref the reference frame's layer output.  The restored row
 * is the next layer's input, so a token reused at one layer may be recomputed at a later one
 * (in gate mode every token is gated at every layer).  Reused keys and values stay the
 * reference's.  The weights follow the base blob (see dv_weights_floats). */
#define DV_FLAG_RESTORE 1u
#define DV_RESTORE_HIDDEN 128   /* hidden width of the restoration MLP */

/* Learned decision layer as the gate (Section 3.3, decision-layer equations).  In gate mode
 * token i of a non-reference frame f is reused at layer l when d_i > tau, where
 *   d_i = w_2 . GELU(W_1 v_i + b_1) + b_2,   v_i = (s_i, t_i, r_I, r_P, r_B2, r_B1),
 *   s_i  cosine of x_f[i] and x_ref[i] (the convention below),
 *   t_i  the class token's attention weight on token i in frame f's layer l-1, averaged over
 *        the heads (1/N at layer 0),
 *   r    one-hot frame type: every non-reference frame references its group's first frame
 *        alone, the role of a P frame, so r = (0, 1, 0, 0);
 * the codec-metadata cue has no input.  tau = 0 is the paper's rule; other finite values move
 * the operating point; -INFINITY and +INFINITY keep their meanings.  GELU is the exact erf
 * form; d is computed in fp32.  The decision is not monotone over layers: every token is gated
 * at every layer, and a reused token's row is the reference's layer output (restored with
 * DV_FLAG_RESTORE).  The weights follow the base blob and the restoration section. */
#define DV_FLAG_DECISION 2u
#define DV_DECISION_HIDDEN 64     /* hidden width of the decision MLP */
#define DV_DECISION_FEATURES 6    /* its input width: s, t and the four frame types */

/* Reordered referencing with past and future references (Section 3.1, frame reordering;
 * Eq. 1 with two references) instead of the star.  The group size must be a multiple of 4.
 * Within a group of G frames the first is the I frame (computed in full); positions 4, 8, ...
 * are P frames referencing the anchor four frames back; between anchors a and a + 4 (the next
 * group's I frame closes the group's last block) the frame at a + 2 is B_dist2, referencing
 * both anchors, and the frames at a + 1 and a + 3 are B_dist1, referencing their neighbours
 * among a, a + 2, a + 4.  A reference past the last frame of the call is absent.  A token's
 * similarity is the larger of its two cosines; when reused, its keys, values and layer output
 * come from the reference that gave it (the past one on a tie).  The decision MLP's type cue is
 * the frame's own type.  Frame indices are those of the call; internal batches also compute
 * the next batch's first frame, so batching does not change results.  With DV_FLAG_RESTORE a
 * reused token's new row is its source token's new row plus its own restoration output (of its
 * input's difference to the source's input); the group size is then at most 60 (chains of
 * sources up to 16 long).  No extra weights. */
#define DV_FLAG_REORDER 4u

typedef struct dv_handle dv_handle;

/* Number of floats the weight blob of `cfg` must hold (0 if cfg is NULL or invalid).
 * The blob holds the ViT backbone of Section 2.3 (and the Section 3.3 MLPs when flagged).
 * Blob layout (fp32, tensors back to back):
 *   W_pe [D,3,p,p], b_pe [D], cls [D], pos [N,D]
 *   per layer: ln1_g [D], ln1_b [D], W_qkv [3D,D], b_qkv [3D], W_o [D,D], b_o [D],
 *              ln2_g [D], ln2_b [D], W_1 [Dm,D], b_1 [Dm], W_2 [D,Dm], b_2 [D]
 *   lnf_g [D], lnf_b [D]
 *   with DV_FLAG_RESTORE, then per layer: W_r1 [R,D], b_r1 [R], W_r2 [D,R], b_r2 [D]
 *   (R = DV_RESTORE_HIDDEN)
 *   with DV_FLAG_DECISION, then per layer: W_d1 [Hd,6], b_d1 [Hd], W_d2 [1,Hd], b_d2 [1]
 *   (Hd = DV_DECISION_HIDDEN; kept in fp32 for every dtype)
 * Linear layers map x -> x W^T + b.  W_qkv rows: Q, then K, then V; heads are
 * contiguous slices of D/H rows within each.  LayerNorm eps is 1e-5. */
size_t dv_weights_floats(const dv_config* cfg);

/* Create a handle for the encoder of Section 2.3 (plus the Section 3.3 layers when flagged):
 * validates cfg, copies the weight blob (`weights`, host,
 * `weights_bytes` bytes, the caller may free it on return) to the device,
 * rounds the matrices to bf16 (nearest, ties to even) when dtype is
 * DV_BF16, and allocates the workspace for max_batch_frames frames together with the stream
 * state of dv_stream_encode (the cached reference, and under DV_FLAG_REORDER the held frames),
 * so that no encode or stream call allocates.  dv_workspace_bytes reports the total.
 * Also looks up, once per device, the static scratch array of dv_encode_noalloc.
 * Synchronous.  Errors: DV_EINVAL (null pointer, wrong blob size, sizes < 1),
 * DV_EUNSUPPORTED (S % p, D % H, head dim, unknown flag bits), DV_ENOMEM (an allocation
 * failed, or the weights and workspace exceed the environment variable DV_MAX_DEVICE_BYTES when
 * it is set -- checked before any device call), DV_EHIP.
 * On error *out is set to NULL. */
int dv_create(const dv_config* cfg, const float* weights, size_t weights_bytes, dv_handle** out);

/* Release a handle and its device memory (synchronises the device first; the lifetime end of
 * the state dv_create made for Section 2.3's encoder).  A NULL handle is accepted. */
int dv_destroy(dv_handle* h);

/* Message of the last error raised on the calling thread ("" if none).  Host-side bookkeeping;
 * no passage of the paper defines it. */
const char* dv_last_error(void);

/* Bytes of device workspace the handle holds (weights excluded): the per-layer batch buffers
 * of layer-wise scheduling and cached memory compaction (Sections 5.1, 5.2) and the stream
 * state (Section 6.3). */
int dv_workspace_bytes(const dv_handle* h, size_t* bytes);

/* Gate mode: the reuse-aware forward of Section 3.3 (similarity cue, Eq. 1; hard gate; token
 * filtration; recompute; token reconstruction) over layer-wise scheduled batches (Section 5.1)
 * with sparse computation compaction (Section 5.3).
 * frames: device fp32 [n_frames, 3, S, S], already normalised.
 * out_embeddings: device fp32 [n_frames, D] (final LayerNorm of the class token).
 * out_masks: device u8 [n_frames, depth, N] (1 = reused; with DV_FLAG_REORDER, 2 = reused
 * from the future reference) or NULL.
 * Frame f's reference is frame G*floor(f/G) (frame indices within this call;
 * a short last group still uses its first frame), or its I/P/B anchors with
 * DV_FLAG_REORDER.  Work is split into internal batches of whole groups, so the
 * result does not depend on max_batch_frames.  tau = -INFINITY turns reuse off (the same kernels run
 * densely, masks all 0); tau = +INFINITY reuses every non-class token of
 * every non-reference frame; a finite tau applies the rule above
 * (tau > 1 reuses nothing, tau <= -1 everything) or, with DV_FLAG_DECISION,
 * the decision MLP's rule d_i > tau.  NaN tau -> DV_EINVAL.
 * Enqueued on `stream`, asynchronous, no host synchronisation.
 * Errors: DV_EINVAL (null handle/frames/embeddings, n_frames < 1,
 * group_size < 1 or > max_batch_frames, NaN tau, group_size not a multiple of 4 with
 * DV_FLAG_REORDER, or above 60 with DV_FLAG_REORDER and DV_FLAG_RESTORE), DV_EHIP. */
int dv_encode(dv_handle* h, const float* frames, int n_frames, int group_size, float tau,
              float* out_embeddings, uint8_t* out_masks, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): dv_encode with its workspace taken from a static
 * device array of DV_SCRATCH_BYTES bytes instead of the handle's.  Same arguments, results and
 * errors as dv_encode (results are bitwise those of dv_encode: they do not depend on the
 * internal batch size).  Frames are encoded in internal batches of as many whole groups as the
 * array holds (at most max_batch_frames); a single group that does not fit is rejected with
 * DV_ENOMEM before anything is launched.  The call allocates nothing and creates no events
 * (stage timing is off for it).  Each device holds one copy of the array for the life of the
 * process, looked up by dv_create; every call on a device uses that one copy, so calls that
 * overlap on one device (other streams, other threads, other handles) race and must be
 * serialised by the caller.  DV_EHIP if the array's address could not be looked up. */
#define DV_SCRATCH_BYTES (128ull << 20)
int dv_encode_noalloc(dv_handle* h, const float* frames, int n_frames, int group_size, float tau,
                      float* out_embeddings, uint8_t* out_masks, hipStream_t stream);

/* Mask-injection mode (Section 3.3 with the hard gate's map M supplied by the caller instead of
 * computed): the reuse map comes from `masks`, device u8
 * [n_frames, depth, N] (nonzero = reuse), instead of the gate.  Entries of
 * class tokens and of reference frames are forced to 0; out_masks (optional)
 * receives the effective map.  Masks need not be monotone over layers: a
 * token reused at layer l holds the reference's row at layer l+1.
 * Other arguments and errors as dv_encode (masks NULL -> DV_EINVAL). */
int dv_encode_masked(dv_handle* h, const float* frames, int n_frames, int group_size,
                     const uint8_t* masks, float* out_embeddings, uint8_t* out_masks,
                     hipStream_t stream);

/* Either mode (masks != NULL selects injection and ignores tau), plus the
 * last layer's full token buffer (the reconstructed tokens of Section 3.3): out_tokens device fp32 [n_frames, N, D]
 * (NULL allowed).  Used to check whole outputs, not only embeddings. */
int dv_encode_tokens(dv_handle* h, const float* frames, int n_frames, int group_size, float tau,
                     const uint8_t* masks, float* out_embeddings, uint8_t* out_masks,
                     float* out_tokens, hipStream_t stream);

/* Streaming (frames arriving in calls of any size; Section 6.3's periodic I frame every G
 * frames, and a group may span calls).  The handle numbers the frames of successive
 * dv_stream_encode calls g = 0, 1, ... since the last dv_stream_reset (or creation); frame g's
 * reference is frame G * floor(g / G), which may have come in an earlier call: the handle then
 * keeps that reference's per-layer input rows and keys/values in a cache ((L+1) N D fp32 plus
 * L N 2D dtype elements, part of the workspace dv_create allocates) instead of recomputing it.  Results
 * are those of one dv_encode_tokens call over all frames of the stream.  frames, masks (NULL:
 * gate mode with tau), out_embeddings, out_masks and out_tokens (both may be NULL) cover this
 * call's frames, with the layouts of dv_encode_tokens.  group_size must stay the same until the
 * next reset.
 * With DV_FLAG_REORDER (the paper's streaming use of reordering, which buffers a few frames):
 * a frame between anchors a and a + 4 (stream indices that are multiples of 4) needs the later
 * anchor, so the frames after the last anchor received so far (at most 3) are held by the
 * handle and encoded by the call that brings their anchor.  A call then outputs the frames it
 * completes, in stream order: the frames held before it, then its own frames up to its last
 * anchor; their number is n_frames + (frames held before) - (frames held after), see
 * dv_stream_held, and the output buffers must have room for n_frames + 3 frames.  A held
 * frame is encoded with the tau of the call that completes it; a stream holding frames must
 * keep to gate mode or to injected maps (DV_EINVAL otherwise); the held frames' maps are kept.
 * dv_stream_flush encodes the held frames as the stream's last.  Results, with the flush, are
 * those of one dv_encode_tokens call over all frames of the stream.  Needs max_batch_frames >
 * group_size; the handle also keeps the held frames' pixels and maps and a staging area for
 * maps (3 frames of pixels, (3 + max_batch_frames) L N bytes).
 * Errors as dv_encode_tokens, plus DV_EINVAL for a changed group_size, a stream left
 * inconsistent by a failed call (reset it), a reordered stream switching between gate mode and
 * injected maps while frames are held, or max_batch_frames <= group_size under reordering.
 * Allocates nothing. */
int dv_stream_encode(dv_handle* h, const float* frames, int n_frames, int group_size, float tau,
                     const uint8_t* masks, float* out_embeddings, uint8_t* out_masks,
                     float* out_tokens, hipStream_t stream);
/* Forget the stream position, the cached reference and any held frames (the memory is kept;
 * Section 6.3's reset of the reference chain). */
int dv_stream_reset(dv_handle* h);
/* Number of frames a reordered stream holds (Section 6, frame reordering in streaming use
 * buffers frames until their later anchor; 0 .. 3; always 0 without DV_FLAG_REORDER), a host
 * value known when the last call returned.  Errors: DV_EINVAL (null handle or n_held). */
int dv_stream_held(const dv_handle* h, int* n_held);
/* End a stream (Section 6.3): encode the held frames (DV_FLAG_REORDER) as its last frames, whose later anchor
 * is absent, with the mode and tau of the last dv_stream_encode call, write their results to
 * out_embeddings, out_masks and out_tokens (the latter two may be NULL; layouts as
 * dv_stream_encode), then reset the stream.  With no held frames only the reset happens.
 * Errors: DV_EINVAL (null handle; null out_embeddings while frames are held), DV_EHIP. */
int dv_stream_flush(dv_handle* h, float* out_embeddings, uint8_t* out_masks, float* out_tokens,
                    hipStream_t stream);

/* Stream compaction of a reuse map on its own (token filtration, Section 3.3;
 * stream compaction across the frames of a batch, Section 5.3).
 * masks: device u8 [n_frames, n_tokens], 1 = reused; entries of reference
 * frames (f % group_size == 0) must be 0 (the caller's contract; reference
 * rows are counted as recomputed whatever they hold).
 * Outputs (device, int32): idx [n_frames*n_tokens] -- the recomputed tokens
 * f*n_tokens+i in frame-major order in idx[0..count); pos
 * [n_frames*n_tokens] -- packed slot of each token, for a reused token the
 * slot of the same token of its reference frame; qoff [n_frames+1] -- first
 * packed slot of each frame, qoff[n_frames] = count; count [1].
 * Errors: DV_EINVAL (null pointer, sizes < 1, n_frames*n_tokens > 2^30), DV_EHIP. */
int dv_compact(const uint8_t* masks, int n_frames, int n_tokens, int group_size, int32_t* idx,
               int32_t* pos, int32_t* qoff, int32_t* count, hipStream_t stream);

/* Stage timing (measurement support; the stages are the steps of Sections 2.3 and 3.3) with
 * HIP events recorded on the encode stream around every
 * launch of the selected stages.  stage_mask: bit s selects stage s (0 = off,
 * DV_PROFILE_ALL = every stage).  While on, every dv_encode* call records;
 * read the totals after synchronising the stream.  dv_profile resets them. */
#define DV_STAGE_PATCH 0
#define DV_STAGE_GATE 1
#define DV_STAGE_COMPACT 2
#define DV_STAGE_LN1 3   /* LN1 is computed by the gate pass: no launches of its own */
#define DV_STAGE_QKV 4
#define DV_STAGE_ATTN 5
#define DV_STAGE_OPROJ 6
#define DV_STAGE_LN2 7
#define DV_STAGE_FC1 8
#define DV_STAGE_FC2 9
#define DV_STAGE_MERGE 10
#define DV_STAGE_FINAL 11
#define DV_STAGE_RESTORE 12   /* the two restoration GEMMs (DV_FLAG_RESTORE) */
#define DV_STAGE_CLS 13       /* class-token attention weights for the decision MLP */
#define DV_NUM_STAGES 14
#define DV_PROFILE_ALL 0x3FFF
int dv_profile(dv_handle* h, unsigned stage_mask);
/* total_ms: summed event time of the stage's launches; launches: how many. */
int dv_profile_read(dv_handle* h, int stage, double* total_ms, long long* launches);

/* Measured MFMA ceiling (measurement support: the roofline of the packed GEMMs of Section 3.3 is
 * also quoted against what the matrix cores sustain on this chip, not only the nominal peak).
 * Enqueues on `stream` one launch of `blocks` blocks of four wavefronts; each wavefront runs
 * `iters` rounds of four independent chains of v_mfma_f32_32x32x16_bf16 on random register
 * operands, with no memory traffic, and stores one float per lane to `sink` (device,
 * blocks*256 floats, caller-owned; the values are meaningless).  *flops (host) receives the
 * FLOPs of the launch; time it with events on `stream`.  Two blocks per compute unit (two
 * wavefronts per SIMD) are resident at once.
 * Errors: DV_EINVAL (NULL sink or flops, blocks outside [1, 2^20], iters < 1), DV_EHIP. */
int dv_mfma_probe(int blocks, int iters, float* sink, double* flops, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* DEJAVU_H */
