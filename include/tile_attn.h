/*
 * tile_attn.h -- C ABI of the gfx950 (MI355X) tile-sparse 3D attention library.
 *
 * Operation (Efficient-vDiT, arXiv 2502.06155, Sec. 3.1 and Sec. 3.3): a video
 * token sequence of S = F * T tokens is flattened frame-major (Sec. 4.1), so
 * token s belongs to latent frame s / T. A frame-level F x F tile mask decides,
 * for each query frame i, which key frames j it attends to. For a query token s
 * of frame i,
 *
 *     out[s] = sum_t softmax_t(scale * <q[s], k[t]>) * v[t]
 *
 * over the key tokens t of the kept frames only; a query frame with no kept key
 * frame produces zeros. Tiles the mask drops are never read or computed (the
 * block skipping of App. B), so work grows with the number of kept tiles, which
 * for the k:(F-k) masks (diagonal plus k global reference frames) is linear in F.
 *
 * Conventions shared by all entry points:
 *   - q, k, v, out are DEVICE pointers to bf16 values (raw 16-bit storage),
 *     contiguous [B, H, S, d] with S = F * T, frame-major tokens, each pointer
 *     16-byte aligned. out must not overlap q, k or v. The caller owns them.
 *   - Accumulation is fp32 (QK^T and PV on bf16 matrix cores, softmax state in
 *     fp32); out is rounded to bf16 with round-to-nearest-even.
 *   - d (head dimension) must be 64, 96 or 128. B, H, F, T >= 1,
 *     F <= TA_MAX_FRAMES, S <= 2^31 - 1; offsets are 64-bit.
 *   - scale must be finite; 1/sqrt(d) is the usual choice. Any sign is allowed.
 *   - stream is a hipStream_t passed as void*; NULL means the null stream. The
 *     call is asynchronous: it enqueues the kernel and returns.
 *   - Argument errors are detected before any HIP call: the status is returned
 *     and nothing is enqueued. A HIP failure returns TA_ERR_HIP; the detail is in
 *     tile_attn_last_error().
 *   - Thread-safe. The first call for a given mask (per device) uploads its
 *     work plan (tile_attn_plan) with a blocking allocation and copy. Device
 *     copies of plans are cached, at most TA_PLAN_CACHE_ENTRIES of them (each
 *     4 * (5 * items + kept entries + 4 * split frames) bytes, plus for a forward
 *     launch's schedule 128 bytes, 16 per part and 12 per query block cut into
 *     parts; a gradient call holds two: the mask's and its transpose's; a forward
 *     plan is cached per launch shape). Beyond that the least recently
 *     used one is evicted; its memory is freed only once no call holds it and
 *     events recorded after every call that used it have completed, so evicting
 *     never waits for a stream. A plan used while its stream is being captured
 *     into a graph is never evicted (the graph may replay at any later time). A
 *     mask whose plan splits heavy query frames also needs a workspace for the
 *     partial results, n_slots * B * max(T, P) * (d + 1) * 4 bytes (n_slots
 *     counts the pieces of all heads), and so does a forward launch whose last
 *     round of workgroups on some XCD would be ragged: where the plan splits no
 *     frame, that round's query blocks are cut into parts over their kept tiles,
 *     n_parts * R * (d + 4) * 4 bytes (R = 256 query rows per block, 128 at
 *     d = 128; n_parts is at most 16 per block cut, and zero when the launch
 *     fills whole rounds, and for video-only calls at d = 64 and 96 whose frames
 *     end on a block of at most 32 rows, which run those blocks last instead).
 *     An MM-DiT forward at d = 64 whose plan splits frames
 *     also uses 256 bytes of work-queue counters, allocated and zeroed
 *     (synchronously) by the first such call on a stream; every call leaves them
 *     zero. The workspace is held per (device, stream). A call that needs more
 *     allocates a larger one (at least 1.5 times the size) and keeps the old one
 *     allocated until process exit, so no enqueued work ever sees its workspace
 *     freed and growing never waits for the stream. Later calls that fit allocate
 *     nothing and do not synchronise, so a warmed-up call can be captured in a
 *     HIP graph.
 *   - The workspace and the counters are found by the stream handle: calls on
 *     one stream share them in stream order, calls on different live streams
 *     never share them. Two cases do share them with work that may still run,
 *     so avoid them: a stream destroyed with calls still pending whose handle a
 *     new stream then receives (synchronise a stream before destroying it), and
 *     a captured graph replayed on another stream while calls run on the stream
 *     it was captured on (the graph holds that stream's workspace and counters).
 */
#ifndef TILE_ATTN_H
#define TILE_ATTN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TA_MAX_FRAMES 1024
#define TA_PLAN_CACHE_ENTRIES 256
#define TA_NOALLOC_PLAN_WORDS 65536
#define TA_NOALLOC_PARTIAL_BYTES (64u << 20)

typedef enum {
  TA_OK = 0,
  TA_ERR_NULL_PTR = 1,  /* a required pointer is NULL */
  TA_ERR_BAD_SHAPE = 2, /* B, H, F, T out of range, S or the grid overflows */
  TA_ERR_HEAD_DIM = 3,  /* d is not 64, 96 or 128 */
  TA_ERR_BAD_MASK = 4,  /* mask recipe out of range (tile_attn_make_mask) */
  TA_ERR_ALIGN = 5,     /* a tensor pointer is not 16-byte aligned */
  TA_ERR_BAD_SCALE = 6, /* scale is NaN or infinite */
  TA_ERR_OVERLAP = 7,   /* out overlaps q, k or v */
  TA_ERR_HIP = 8        /* a HIP runtime call or the launch failed */
} ta_status;

/* Mask forms for tile_attn_make_mask. */
typedef enum {
  TA_MASK_COL = 0,  /* query frame i keeps key frame i and every global frame */
  TA_MASK_SYM = 1,  /* TA_MASK_COL, plus every global query frame keeps all frames */
  TA_MASK_DENSE = 2 /* every tile kept (3D full attention) */
} ta_mask_form;

/*
 * Tile-sparse attention forward (Sec. 3.3; kernel-only benchmark of Sec. 4.2.1:
 * inputs query, key, value and mask, output the attention output).
 *
 * tile_mask: HOST pointer to F*F bytes, row-major [query_frame][key_frame];
 * nonzero = tile kept. It is read during the call only. The mask is
 * authoritative: no diagonal is added.
 */
int tile_attn_fwd(const void* q, const void* k, const void* v, void* out,
                  int B, int H, int F, int T, int d,
                  const uint8_t* tile_mask, float scale, void* stream);

/*
 * Tile-sparse attention forward with one mask per head and an optional row
 * log-sum-exp. The layer-wise search of Sec. 3.3 (Alg. 1) gives each layer, and
 * the heads within it, their own k:(F-k) pattern; the log-sum-exp is what a
 * merge of partial results or a backward pass needs.
 *
 * tile_masks: HOST pointer to n_masks * F * F bytes, mask after mask, each
 *   row-major [query_frame][key_frame], nonzero = kept; n_masks == 1 shares one
 *   mask across all heads (tile_attn_fwd), n_masks == H gives mask h to head h.
 *   Read during the call only.
 * lse: DEVICE pointer to fp32 [B, H, S], 4-byte aligned, or NULL. Receives for each
 *   query token the natural-log log-sum-exp of scale * <q, k_t> over its kept keys
 *   t (computed from the bf16-rounded weights that also weight V), and -inf for a
 *   query frame that keeps nothing. Must not overlap q, k, v or out.
 * Errors: those of tile_attn_fwd, plus TA_ERR_BAD_MASK when n_masks is neither 1
 *   nor H, TA_ERR_ALIGN for a misaligned lse and TA_ERR_OVERLAP when lse overlaps
 *   a tensor.
 */
int tile_attn_fwd_heads(const void* q, const void* k, const void* v, void* out,
                        int B, int H, int F, int T, int d,
                        const uint8_t* tile_masks, int n_masks, float scale,
                        float* lse, void* stream);

/*
 * The MM-DiT form (Sec. 4.3 and App. E: CogVideoX concatenates text tokens with
 * the video tokens and the sparse mask covers only the video-video part). Each
 * (batch, head) sequence holds P text tokens first, then the F * T video tokens
 * frame-major: S = P + F * T. A text query attends to all S tokens; a query of
 * video frame i attends to the P text tokens and to the tokens of the video frames
 * its mask row keeps.
 *
 * q, k, v, out: DEVICE bf16 [B, H, P + F*T, d], 16-byte aligned. P >= 0 (P = 0
 *   is tile_attn_fwd_heads). tile_masks, n_masks: F x F video masks as for
 *   tile_attn_fwd_heads. lse: as for tile_attn_fwd_heads over the S rows, or NULL.
 *   The text queries keep every segment, so their work is split into pieces like
 *   any heavy query frame (tile_attn_plan of the (F+1) x (F+1) mask whose last row
 *   and column, the text, are all ones).
 * Errors: those of tile_attn_fwd_heads; TA_ERR_BAD_SHAPE also for P < 0 or
 *   P + F*T > 2^31 - 1.
 */
int tile_attn_fwd_mmdit(const void* q, const void* k, const void* v, void* out,
                        int B, int H, int F, int T, int P, int d,
                        const uint8_t* tile_masks, int n_masks, float scale,
                        float* lse, void* stream);

/*
 * Gradients of tile-sparse attention (the op the sparse student of Sec. 3.4 is
 * trained through). With P[s,t] = exp(scale * <q[s], k[t]> - lse[s]) over the kept
 * pairs, dP[s,t] = <dout[s], v[t]>, delta[s] = <dout[s], out[s]> and
 * dS = P * (dP - delta):
 *     dq[s] = scale * sum_t dS[s,t] k[t],  dk[t] = scale * sum_s dS[s,t] q[s],
 *     dv[t] = sum_s P[s,t] dout[s],
 * sums over kept pairs only: keys of frames no query frame keeps get zero dk and
 * dv, queries of frames that keep nothing get zero dq. Dropped tiles are never
 * read.
 *
 * q, k, v: the forward's inputs; out, lse: what tile_attn_fwd_heads returned for
 *   them with the same masks and scale (out bf16 [B, H, S, d], lse fp32 [B, H, S],
 *   DEVICE). dout: DEVICE bf16 [B, H, S, d], the gradient of out.
 * dq, dk, dv: DEVICE bf16 [B, H, S, d] outputs, fully written (rounded to bf16,
 *   RNE, from fp32 sums). They must not overlap each other or any input.
 * tile_masks, n_masks: as for tile_attn_fwd_heads. All bf16 tensors 16-byte
 *   aligned, lse 4-byte aligned.
 * Workspace: B*H*S*8 bytes for the base-2 lse and delta, plus fp32 partials for
 *   frames the plan splits (the query side plans the mask, the key side its
 *   transpose, each as tile_attn_plan describes), held per (device, stream) like
 *   the forward's.
 * Errors: those of tile_attn_fwd_heads (TA_ERR_NULL_PTR also for out, dout, lse,
 *   dq, dk, dv; TA_ERR_OVERLAP when an output overlaps an input or another
 *   output).
 */
int tile_attn_bwd(const void* q, const void* k, const void* v, const void* out,
                  const void* dout, const float* lse, void* dq, void* dk, void* dv,
                  int B, int H, int F, int T, int d,
                  const uint8_t* tile_masks, int n_masks, float scale, void* stream);

/*
 * Gradients of the MM-DiT form (tile_attn_fwd_mmdit): the same chain rule over the
 * query-key pairs that form keeps (text rows and text columns dense, the video masks
 * on the video-video part), for training a sparse MM-DiT student (App. E applies
 * the method's distillation to CogVideoX). Tensors are [B, H, P + F*T, d] with the
 * P text tokens first; out and lse come from tile_attn_fwd_mmdit with the same
 * masks and scale. P = 0 is tile_attn_bwd. Every key is kept by the text queries,
 * so the key side plans the transposed (F+1) x (F+1) mask, whose text row is
 * split. Errors: those of tile_attn_bwd; TA_ERR_BAD_SHAPE also for P < 0.
 */
int tile_attn_bwd_mmdit(const void* q, const void* k, const void* v, const void* out,
                        const void* dout, const float* lse, void* dq, void* dk, void* dv,
                        int B, int H, int F, int T, int P, int d,
                        const uint8_t* tile_masks, int n_masks, float scale, void* stream);

/*
 * Dense control: 3D full attention (every tile kept, the "full" rows of
 * tab:kernel_time). Runs the same kernel as tile_attn_fwd with an all-ones
 * mask, so its output is bit-identical to tile_attn_fwd with that mask.
 */
int dense_attn_fwd(const void* q, const void* k, const void* v, void* out,
                   int B, int H, int F, int T, int d, float scale, void* stream);

/*
 * Build a k:(F-k) mask (Sec. 3.3): the main diagonal plus k global reference
 * frames chosen uniformly, frames 0, s, 2s, ... below F with s = ceil(F / k)
 * (fewer than k frames when the stride overshoots). form selects how the
 * reference frames are kept (ta_mask_form). With TA_MASK_SYM this placement
 * reproduces every sparsity printed in tab:kernel_time.
 *
 * mask_out: HOST buffer of F*F bytes, written row-major with 0/1.
 * Errors: TA_ERR_NULL_PTR, TA_ERR_BAD_SHAPE (F outside 1..TA_MAX_FRAMES),
 * TA_ERR_BAD_MASK (k outside 0..F or unknown form). Touches no GPU.
 */
int tile_attn_make_mask(int F, int k, int form, uint8_t* mask_out);

/*
 * The compact kept-tile list the kernels walk instead of the dense mask
 * (App. B: masked blocks are skipped and the full mask is never materialised).
 *
 * row_ptr: HOST int32[F+1]; kept key frames of query frame i are
 *   cols[row_ptr[i] .. row_ptr[i+1]), ascending.
 * cols: HOST uint16[F*F] (capacity F*F; the first *nnz entries are written).
 * order: HOST uint16[F]; query frames by descending kept-tile count (ties by
 *   frame index), the order in which work is dispatched. May be NULL.
 * nnz: HOST int, receives the number of kept tiles.
 * Errors: TA_ERR_NULL_PTR, TA_ERR_BAD_SHAPE. Touches no GPU.
 */
int tile_attn_compact(const uint8_t* tile_mask, int F, int32_t* row_ptr,
                      uint16_t* cols, uint16_t* order, int* nnz);

/*
 * The work plan the kernels execute for a mask (host only, touches no GPU). Every
 * query frame is one work item over its kept key frames, except that a frame
 * keeping more than twice the mean number of kept frames per row (rounded up) is
 * split into up to 32 items of about that mean size, whose partial results
 * (slot >= 0) a merge pass combines by their log-sum-exp: one heavy row (the
 * global query frames of the symmetric mask keep every frame) then no longer
 * sets the critical path of the launch. The pieces of a split frame cover its
 * kept list contiguously and in order. tile_attn_fwd falls back to the unsplit
 * plan when the partial results would need more than 2 GiB.
 *
 * items: HOST int32[4 * cap]; item i is {query frame, first kept entry (index into
 *   the row-after-row kept list of tile_attn_compact), number of kept entries,
 *   slot or -1}, items ordered by descending kept count (ties keep frame order).
 * n_items, n_slots: HOST ints receiving the item and partial-slot counts.
 * Errors: TA_ERR_NULL_PTR, TA_ERR_BAD_SHAPE (F out of range, or cap < n_items; the
 * counts are still written).
 */
int tile_attn_plan(const uint8_t* tile_mask, int F, int32_t* items, int cap, int* n_items,
                   int* n_slots);

/*
 * tile_attn_fwd_heads for callers that cannot allocate device memory: code being
 * captured into a HIP graph, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments and errors as tile_attn_fwd_heads, but the call allocates
 * nothing (no hipMalloc, hipFree or allocating library routine): its work plan and
 * the partial results of split query frames live in one static device array per GPU,
 * TA_NOALLOC_PLAN_WORDS int32 words for the plan plus TA_NOALLOC_PARTIAL_BYTES for
 * the partials (about 64.25 MiB), held from the library's first use on a GPU until
 * the process ends. The plan reaches the array by value, in the arguments of small
 * store kernels enqueued on `stream`, so the call only enqueues kernels and reads no
 * host memory after it returns.
 *
 * It never cuts a launch's last round into parts, so where tile_attn_fwd_heads does,
 * the two agree up to rounding order only (bit for bit otherwise).
 *
 * Every call on one GPU shares that GPU's array, so calls whose execution overlaps
 * on one GPU (on different streams, or graphs replayed concurrently) race: order
 * them on one stream. A mask whose split plan needs more partial space than the
 * array holds runs unsplit (each heavy query frame as one work item; same results up
 * to rounding order, the heavy rows then set the launch's critical path).
 * Errors: those of tile_attn_fwd_heads; TA_ERR_BAD_SHAPE also when the plan exceeds
 * TA_NOALLOC_PLAN_WORDS words (about 5 * H * F + nnz of all masks).
 */
int tile_attn_fwd_heads_noalloc(const void* q, const void* k, const void* v, void* out,
                                int B, int H, int F, int T, int d,
                                const uint8_t* tile_masks, int n_masks, float scale,
                                float* lse, void* stream);

/*
 * Occupancy of the plan cache (all devices): *live receives the number of cached
 * plans (at most TA_PLAN_CACHE_ENTRIES, plus any held by calls in progress or pinned
 * by graph capture), *retired the number of evicted plans whose memory waits for
 * their last kernels to finish. Frees the retired plans whose work is done first.
 * Host only; TA_ERR_NULL_PTR for a NULL argument.
 */
int tile_attn_plan_cache_stats(int* live, int* retired);

/* Static text for a status code. */
const char* tile_attn_status_string(int status);

/* Detail of the last error on the calling thread (empty string if none). */
const char* tile_attn_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* TILE_ATTN_H */
