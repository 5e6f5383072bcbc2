/*
 * mv.h -- C ABI of libmv: view-masked causal attention and the fused LM-head
 * token log-prob for scoring a memory-compressed agent trajectory under the
 * live views it was decoded from (MemoryWalker, arXiv 2609.00865), on AMD
 * MI355X (gfx950).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Status: every call returns mv_status.  On failure nothing is launched,
 *    no output is written, and mv_last_error() holds a message for the calling
 *    thread.  No C++ exception crosses this boundary.
 *  - Device memory: the library never allocates device memory.  Every device
 *    buffer (inputs, outputs, the uploaded mask, workspaces) is allocated by
 *    the caller and sized with the *_bytes queries.  Device pointers must be
 *    16-byte aligned and live on the current HIP device.
 *  - Host memory: host arrays owned by a mv_view_mask are freed by
 *    mv_view_mask_free.  Input arrays passed by the caller are only read
 *    during the call.
 *  - Streams: device work is enqueued asynchronously on the given stream
 *    (0 = the null stream).  Host-only calls are synchronous.
 *  - Element types: "bf16" is IEEE bfloat16 stored as 16-bit words; fp32 is
 *    IEEE binary32.  Arithmetic: bf16 matrix products with fp32 accumulation;
 *    softmax statistics in fp32; one round-to-nearest-even to bf16 per
 *    stored bf16 output.
 *  - Thread safety: calls on distinct mask objects are independent; a mask
 *    object must not be used while it is being uploaded or freed.
 */
#ifndef MV_H_
#define MV_H_

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MV_OK = 0,
  MV_ERR_INVALID_ARG = 1,  /* null pointer, negative size, misaligned buffer   */
  MV_ERR_BAD_RECORD = 2,   /* eviction record that no rollout could produce    */
  MV_ERR_SHAPE = 3,        /* tensor shapes inconsistent with each other        */
  MV_ERR_UNSUPPORTED = 4,  /* valid request outside what the kernels implement  */
  MV_ERR_WORKSPACE = 5,    /* workspace or mask buffer smaller than required    */
  MV_ERR_HIP = 6,          /* a HIP runtime call or kernel launch failed        */
  MV_ERR_STATE = 7         /* object not ready (e.g. mask not uploaded)         */
} mv_status;

/* Static name of a status code. */
const char* mv_status_string(mv_status s);
/* Message describing the last failure on the calling thread ("" if none). */
const char* mv_last_error(void);
/* Library ABI version: (major << 16) | minor. */
int32_t mv_version(void);

/* ---------------------------------------------------------------------------
 * Eviction records and the view mask
 *
 * A rollout's record is its physical token sequence (the depth-first tape
 * H_full) plus the ordered edits (J_k, E_k) (Appendix E.1, "one record per
 * rollout"; Definition "trajectory tree", Appendix B.1).  The live view of row
 * i is the physical prefix with exactly the edits fired by then applied
 * (Eq. "live-view", Section 3.2).  Positions are physical rows; the logits
 * for token y_t come from row t-1, and edit k is applied before row J_k is
 * evaluated: rows < J_k see E_k, rows >= J_k do not (this reproduces the
 * per-leaf prefixes of Table "running-prefixes").
 *
 * Equivalently every key j has the lifetime [j, omega(j)) of Eq.
 * "4d-mask-def" (Section 4.2), with omega(j) = J_k if j is in E_k and the end
 * of its trajectory otherwise: row i sees key j iff j <= i < omega(j).  A key
 * that a later edit restores (R_k) gains further intervals [J_k, next death);
 * row i sees it iff i lies in one of them.  Several trajectories are packed
 * back to back; a row never sees another trajectory's keys.
 * ------------------------------------------------------------------------ */
typedef struct {
  int32_t begin, end;            /* half-open physical positions [begin, end) */
} mv_span;

typedef struct {
  int32_t junction;              /* J_k: first row evaluated under the post-edit view */
  int32_t n_evict;               /* number of spans in E_k (0 allowed)               */
  const mv_span* evict;          /* E_k: sorted, disjoint spans inside
                                    [trajectory begin, junction); every token
                                    must still be live when the edit fires     */
  mv_span summary;               /* metadata only (begin == end: none); summary
                                    tokens are ordinary keys born at their row;
                                    must lie in the trajectory and not meet E_k */
  int32_t n_restore;             /* number of spans in R_k (0: a plain eviction)   */
  const mv_span* restore;        /* R_k: sorted, disjoint spans of tokens evicted by
                                    earlier edits and not yet restored, live again
                                    from row J_k on at their own positions (an
                                    offload / retrieve memory: a key may leave the
                                    view and re-enter, Appendix E); must not meet E_k */
} mv_edit;

typedef struct {
  int32_t begin, end;            /* physical rows of this trajectory             */
  int32_t n_edits;
  const mv_edit* edits;          /* strictly increasing junctions, begin < J < end */
} mv_trajectory;

typedef struct mv_view_mask mv_view_mask;   /* opaque */

typedef struct {
  int64_t visible_pairs;         /* P = sum_j (omega(j) - j): visible (row, key) pairs */
  int32_t total_tokens;
  int32_t max_view;              /* largest |View(i)|                                 */
  int32_t n_segments;            /* maximal runs of consecutive keys sharing omega    */
  int32_t tiles_full;            /* 128-row x 64-key tiles computed without masking  */
  int32_t tiles_partial;         /* tiles computed with the per-element predicate    */
  int32_t tiles_skipped;         /* causal tiles holding no visible pair              */
  int32_t bwd_items;             /* key-tile work items of the dK/dV pass             */
  int32_t bwd_partial_slots;     /* fp32 partial tiles the dK/dV pass reduces         */
  int32_t n_leaves;              /* diverging leaves (see mv_view_mask_leaves)        */
  int64_t fwd_tile_pairs;        /* (row, key) pairs of the forward / dQ tiles run    */
  int64_t bwd_tile_pairs;        /* (row, key) pairs of the dK/dV tiles run           */
} mv_mask_stats;

/* Which conditioning a mask encodes. */
enum {
  MV_VIEW_LIVE = 0,   /* the live view of every row (Eq. "live-view"): the exact walk */
  MV_VIEW_FINAL = 1   /* the final compressed walk (Eq. "live-vs-final"): every edit
                         applied to every row; an evicted key is seen by its own row
                         only.  This is the student conditioning of SDCC (Section 5.1)
                         and the Naive-Compressed baseline (Section 3.3, Pitfall A). */
};

/*
 * Build the key-lifetime array omega (Eq. "4d-mask-def") and the block-sparse
 * tile schedules of the attention passes from the eviction records (host only,
 * synchronous).  trajs[0..n_traj) must tile [0, total_tokens) in order.
 * Errors: MV_ERR_INVALID_ARG (null/size), MV_ERR_BAD_RECORD (junction out of
 * range or not increasing, span outside [begin, junction), overlapping spans,
 * a token evicted twice, a summary meeting E_k).  *out is owned by the caller
 * and released with mv_view_mask_free.
 */
mv_status mv_build_view_mask(const mv_trajectory* trajs, int32_t n_traj,
                             int32_t total_tokens, mv_view_mask** out);

/*
 * As mv_build_view_mask, with the tile shape of the forward / dQ schedule
 * named: tile_q query rows x tile_k keys.  The kernels are compiled for
 * MV_TILE_Q x MV_TILE_K (the dK/dV pass walks 128-key tiles in 64-row
 * blocks); any other shape is refused with MV_ERR_UNSUPPORTED before anything
 * is built, so a caller that assumes a tiling learns at once that it differs.
 */
#define MV_TILE_Q 128
#define MV_TILE_K 64
mv_status mv_build_view_mask_tiled(const mv_trajectory* trajs, int32_t n_traj,
                                   int32_t total_tokens, int32_t tile_q, int32_t tile_k,
                                   mv_view_mask** out);

/* As mv_build_view_mask, for kind MV_VIEW_LIVE or MV_VIEW_FINAL. */
mv_status mv_build_view_mask_kind(const mv_trajectory* trajs, int32_t n_traj,
                                  int32_t total_tokens, int32_t kind, mv_view_mask** out);

/*
 * The diverging leaves of the record (Definition "trajectory tree", Appendix
 * B.1; the set C of Section 5.1), in position order: tokens t that survive
 * every edit and whose live view differs from their final-walk prefix, i.e.
 * some key before t is evicted by an edit firing at row t or later.  For each:
 * tokens[i] = t; teacher_rows[i] = t - 1 (the row that predicted t under its
 * live view); student_rows[i] = the last surviving row before t (the row that
 * predicts t on the final compressed walk).  For the running example of
 * Section 3.2 these are y6, y7, y9, y10, y12 (Table "running-prefixes").
 * Host arrays of `capacity` entries; *n_out receives the count.  Passing
 * capacity 0 and null arrays only queries the count.
 */
mv_status mv_view_mask_leaves(const mv_view_mask* m, int32_t* tokens, int32_t* teacher_rows,
                              int32_t* student_rows, int32_t capacity, int32_t* n_out);

/* Bytes of device memory the uploaded mask needs. */
size_t mv_view_mask_device_bytes(const mv_view_mask* m);

/*
 * Copy the mask to a caller-owned device buffer (>= device_bytes, 256-byte
 * aligned) on `stream`; the mask keeps the pointer, so the buffer must outlive
 * every attention call using it.  Uploading again re-targets the mask.
 */
mv_status mv_view_mask_upload(mv_view_mask* m, void* dev_buf, size_t bytes,
                              hipStream_t stream);

mv_status mv_view_mask_stats(const mv_view_mask* m, mv_mask_stats* out);

/* Copy omega (int32[total_tokens], host memory) out of the mask: for every
 * key the end of its first live interval. */
mv_status mv_view_mask_death(const mv_view_mask* m, int32_t* host_out);

/* The further live intervals of keys that edits restore: iv_ptr (int32
 * [total_tokens + 1], nullable) gets, per key, the range of its entries, and
 * iv (int32 [2 * capacity], nullable) the (begin, end) row pairs in time
 * order; *n_out receives the number of intervals.  Host only. */
mv_status mv_view_mask_intervals(const mv_view_mask* m, int32_t* iv_ptr, int32_t* iv,
                                 int32_t capacity, int32_t* n_out);

/*
 * Write the visibility bits the attention kernels act on for rows
 * [row_begin, row_end): bit (j % 32) of word (i - row_begin) * ceil(T/32) + j/32
 * is 1 iff the forward tile schedule visits key j for row i and the shared
 * predicate admits it.  Device variant: dev_bits is device memory, enqueued on
 * `stream` (mask must be uploaded).  Host variant: the same schedule walk and
 * predicate on the CPU.  Both exist so that the schedule and the predicate can
 * be checked bit-exactly against an independent replay of the record.
 */
mv_status mv_view_mask_materialize(const mv_view_mask* m, int32_t row_begin,
                                   int32_t row_end, uint32_t* dev_bits,
                                   hipStream_t stream);
mv_status mv_view_mask_materialize_host(const mv_view_mask* m, int32_t row_begin,
                                        int32_t row_end, uint32_t* host_bits);

void mv_view_mask_free(mv_view_mask* m);

/* ---------------------------------------------------------------------------
 * Branch-replicated packing (Appendix G; the branch layers of Appendix B.1,
 * forwarded as in Section 4.1) for exact multi-layer scoring.
 *
 * Each branch layer k of a trajectory (rows [J_k, J_{k+1})) becomes one
 * segment of a packed stream: the keys live just before J_k in physical
 * order, then the layer's rows.  Under the block-diagonal causal mask every
 * packed row of a layer sees exactly its live view at every depth of a
 * model, and position ids restart per segment, so every copy carries the
 * position its token had in the live context (rotary phases match the
 * rollout).  Per slot: src (physical token copied), pos (index inside its
 * segment), owner (1 for the layer's own rows, which carry their loss; 0 for
 * trunk copies), target (the physical row whose token the slot predicts:
 * src + 1 for owner slots that are not their trajectory's last row, else -1).
 * The packed length is the sum of the layers' lengths, >= total_tokens.
 * Host construction is synchronous; the record rules and errors are those of
 * mv_build_view_mask.
 * ------------------------------------------------------------------------ */
typedef struct mv_branch_pack mv_branch_pack;   /* opaque */

typedef struct {
  int32_t total_tokens;   /* physical rows L                                  */
  int32_t n_packed;       /* packed slots N                                   */
  int32_t n_segments;     /* branch layers over all trajectories              */
  int32_t max_copies;     /* most copies of one physical token                */
  int64_t causal_pairs;   /* visible (row, key) pairs of the mask: for the
                             replicated packing sum over segments of l (l+1)/2 */
} mv_pack_stats;

mv_status mv_build_branch_pack(const mv_trajectory* trajs, int32_t n_traj,
                               int32_t total_tokens, mv_branch_pack** out);

/*
 * LogitTree with shared-trunk KV (Section 4.1: the K+1 branch forwards, whose
 * shared trunk is cached rather than replicated).  Consecutive branch
 * sequences S_{k-1} and S_k agree on their first d_k tokens (up to the first
 * token edit k removes), at the same positions, so those tokens' keys and
 * values are the same at every layer.  Segment k of this packing holds only
 * S_k[d_k:] (segment 0 all of S_0); its rows read the shared prefix from the
 * slots of earlier segments.  The mask (mv_branch_pack_mask) gives every slot
 * one lifetime: the record over the packed stream whose edit at the first
 * slot of segment k evicts the slots holding S_{k-1}[d_k:].  pos is the
 * token's index in its branch sequence (positions restart per branch), owner
 * and target as above; causal_pairs holds the mask's visible pairs.  The
 * result is exact through a stack of layers, like the replicated packing,
 * with each shared prefix computed once.
 */
mv_status mv_build_shared_trunk_pack(const mv_trajectory* trajs, int32_t n_traj,
                                     int32_t total_tokens, mv_branch_pack** out);
mv_status mv_branch_pack_stats(const mv_branch_pack* p, mv_pack_stats* out);
/* Host copies of the layout; every array is optional (null: skipped).
 * src, pos, target: int32 [n_packed]; owner: uint8 [n_packed];
 * seg_begin: int32 [n_segments + 1] (first slot of each segment, then N). */
mv_status mv_branch_pack_layout(const mv_branch_pack* p, int32_t* src, int32_t* pos,
                                uint8_t* owner, int32_t* target, int32_t* seg_begin);
/* The block-diagonal causal mask over the packed stream (each segment a
 * trajectory without edits), owned by the pack: upload it and pass it to the
 * attention entry points like any mask; never free it separately. */
mv_view_mask* mv_branch_pack_mask(mv_branch_pack* p);
/* Device bytes of the layout arrays (src, pos and the per-token copy lists),
 * not counting the mask's own buffer. */
size_t mv_branch_pack_device_bytes(const mv_branch_pack* p);
/* Copy the layout to a caller-owned device buffer (256-byte aligned) that
 * must outlive every call using it; as mv_view_mask_upload. */
mv_status mv_branch_pack_upload(mv_branch_pack* p, void* dev_buf, size_t bytes,
                                hipStream_t stream);
void mv_branch_pack_free(mv_branch_pack* p);

/* out[slot, :] = in[src[slot], :]: bf16 rows of `width` elements (width % 8
 * == 0), in [total_tokens, width], out [n_packed, width]. */
mv_status mv_pack_rows(const mv_branch_pack* p, const void* in, int32_t width, void* out,
                       hipStream_t stream);
/* The adjoint of mv_pack_rows: out[t, :] = sum over the copies of token t, in
 * increasing slot order, of in[slot, :] (fp32 sums), stored as bf16
 * (out_fp32 == 0) or fp32.  Deterministic. */
mv_status mv_unpack_rows_sum(const mv_branch_pack* p, const void* in, int32_t width,
                             int32_t out_fp32, void* out, hipStream_t stream);
/* Rotary embedding of x [n_packed, n_heads, head_dim] (bf16) by each slot's
 * position id: pairs (i, i + head_dim/2) rotate by pos * theta^(-2i/head_dim)
 * (angles in double precision, rotation in fp32, one rounding to bf16).
 * direction +1 applies the rotation, -1 its inverse (which is also its
 * backward).  out may alias x.  head_dim even, <= 256. */
mv_status mv_rope(const mv_branch_pack* p, const void* x, int32_t n_heads, int32_t head_dim,
                  float theta, int32_t direction, void* out, hipStream_t stream);

/* The gather with the rotary embedding fused into it (Appendix G: each
 * branch's positions restart from its own prefix): out[slot] =
 * R(pos[slot]) in[src[slot]], in bf16 [total_tokens, n_heads, head_dim], out
 * bf16 [n_packed, n_heads, head_dim]; one pass instead of mv_pack_rows then
 * mv_rope.  Angles in fp64 (reduced to [-pi, pi] there), their cosine and
 * sine and the rotation in fp32, one rounding to bf16.  head_dim a multiple
 * of 16, <= 256; out must not alias in. */
mv_status mv_pack_rows_rope(const mv_branch_pack* p, const void* in, int32_t n_heads,
                            int32_t head_dim, float theta, void* out, hipStream_t stream);
/* The adjoint of mv_pack_rows_rope: out[t] = sum over the copies of token t,
 * in increasing slot order, of R(pos[slot])^T in[slot] (the inverse rotation
 * of each copy's gradient, summed in fp32, rounded once), stored as bf16
 * (out_fp32 == 0) or fp32 [total_tokens, n_heads, head_dim]; one pass instead
 * of mv_rope (direction -1) then mv_unpack_rows_sum.  Deterministic.
 * head_dim a multiple of 16, <= 256; out must not alias in. */
mv_status mv_unpack_rows_sum_rope(const mv_branch_pack* p, const void* in, int32_t n_heads,
                                  int32_t head_dim, float theta, int32_t out_fp32, void* out,
                                  hipStream_t stream);

/* ---------------------------------------------------------------------------
 * View-masked attention (Section 4.2, the packed single forward; its
 * equivalence with one causal forward per branch is Theorem "hard_equiv",
 * Section 4.3 and Appendix C.3).
 *
 * Layouts (row-major, bf16): Q, O, dO, dQ are [total_tokens, n_heads_q,
 * head_dim]; K, V, dK, dV are [total_tokens, n_heads_kv, head_dim].  Query
 * head h reads KV head h / (n_heads_q / n_heads_kv).  LSE is fp32
 * [n_heads_q, total_tokens], natural log.  Q and K are taken as given
 * (already position-encoded).  head_dim in {64, 128}; each tensor under
 * 4 GiB (total_tokens * n_heads_q * head_dim * 2 bytes < 2^32).
 * ------------------------------------------------------------------------ */
typedef struct {
  int32_t total_tokens;          /* must equal the mask's                          */
  int32_t n_heads_q, n_heads_kv; /* n_heads_q % n_heads_kv == 0                    */
  int32_t head_dim;              /* 64 or 128                                      */
  float softmax_scale;           /* <= 0 selects 1/sqrt(head_dim)                  */
} mv_attn_shape;

/*
 * O_i = sum_{j in View(i)} softmax_j(scale * q_i.k_j) v_j and
 * LSE_i = log sum_{j in View(i)} exp(scale * q_i.k_j), for every row and head.
 * Tiles with no visible pair are skipped; tiles that are entirely visible skip
 * the per-element predicate.
 */
mv_status mv_attn_fwd(const mv_view_mask* m, const mv_attn_shape* shape,
                      const void* q, const void* k, const void* v,
                      void* o, float* lse, hipStream_t stream);

/* Workspace bytes of mv_attn_bwd (row statistics and fp32 dK/dV partials). */
size_t mv_attn_bwd_workspace_bytes(const mv_view_mask* m, const mv_attn_shape* shape);

/*
 * Gradients of sum_i <dO_i, O_i> with respect to Q, K and V under the same
 * views, from the forward's O and LSE: one backward for the whole trajectory
 * (the 4D method's single backward, Section 4.3 "Cost and deployment splits").
 * dQ, dK, dV are fully overwritten.  Deterministic: no atomics.
 */
mv_status mv_attn_bwd(const mv_view_mask* m, const mv_attn_shape* shape,
                      const void* q, const void* k, const void* v,
                      const void* o, const void* dout, const float* lse,
                      void* dq, void* dk, void* dv,
                      void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * backward as mv_attn_bwd, with its workspace replaced by a static scratch
 * array of MV_ATTN_BWD_NOALLOC_SCRATCH_BYTES that the library keeps on each
 * GPU it runs on until the process ends.  The caller still passes every input
 * and output.  A call whose workspace (mv_attn_bwd_workspace_bytes) exceeds
 * the scratch is refused with MV_ERR_WORKSPACE before anything is enqueued.
 * No device memory is allocated or freed, and no events are created (the
 * profiling switch does not apply).  The first call on a device looks up the
 * scratch's address there (a runtime query, once per device).  All calls on
 * one GPU share its scratch: calls that overlap in time on one GPU (other
 * streams, other threads) race and must be serialised by the caller.  Results
 * are bit-identical to mv_attn_bwd's.
 */
#define MV_ATTN_BWD_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

mv_status mv_attn_bwd_noalloc(const mv_view_mask* m, const mv_attn_shape* shape,
                              const void* q, const void* k, const void* v,
                              const void* o, const void* dout, const float* lse,
                              void* dq, void* dk, void* dv, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Fused LM-head token log-prob, importance ratio and clip.
 *
 * z_t = W h_t is never stored.  logp_t = z_{t,y_t} - logsumexp_v z_tv is the
 * log-prob the training pass recomputes under the live view (the left term
 * of Eq. "logdiff", Section 3.1); ratio_t = exp(logp_t - logp_old_t) and
 * clipped_t = clamp(ratio_t, 1 - eps_low, 1 + eps_high) are the GRPO
 * importance ratio and its clip (Appendix C, "Pitfall A, RL view";
 * Appendix F).  target[t] == -1 marks a token without loss: logp 0, ratio 1,
 * clipped 1, zero gradient.  Targets should lie in [-1, vocab); an id outside
 * that range is never used as an index: the kernels treat its token as one
 * without loss and count it in the workspace's status word, which
 * mv_token_logprob_bad_targets reads back.
 *
 * Layouts: hidden bf16 [n_tokens, hidden]; weight bf16 [vocab, hidden];
 * target int32 [n_tokens]; per-token fp32 vectors [n_tokens].
 * Supported: hidden % 64 == 0.
 * ------------------------------------------------------------------------ */
typedef struct {
  int32_t n_tokens, hidden, vocab;
  float eps_low, eps_high;       /* clip range (e.g. 0.2 / 0.2, or 0.2 / 0.28)      */
} mv_logprob_shape;

size_t mv_token_logprob_workspace_bytes(const mv_logprob_shape* shape);

/*
 * logp and lse are required; ratio and clipped are written iff logp_old is
 * non-null (then both must be non-null).
 */
mv_status mv_token_logprob(const mv_logprob_shape* shape, const void* hidden,
                           const void* weight, const int32_t* target,
                           const float* logp_old, float* logp, float* ratio,
                           float* clipped, float* lse, void* workspace,
                           size_t workspace_bytes, hipStream_t stream);

size_t mv_token_logprob_bwd_workspace_bytes(const mv_logprob_shape* shape);

/*
 * dhidden_t = dlogp_t * (W[y_t] - sum_v softmax(z_t)_v W[v])  (bf16 out), from
 * the forward's lse; logits are recomputed, never read back.
 */
mv_status mv_token_logprob_bwd(const mv_logprob_shape* shape, const void* hidden,
                               const void* weight, const int32_t* target,
                               const float* lse, const float* dlogp, void* dhidden,
                               void* workspace, size_t workspace_bytes,
                               hipStream_t stream);

/*
 * Number of target ids outside [-1, vocab) that the last mv_token_logprob or
 * mv_token_logprob_bwd call on `workspace` met (every such token was scored
 * as one without loss).  Waits for the stream's work, then copies one word
 * to *host_count.  The count belongs to the workspace: a later call that
 * uses the same workspace resets it.
 */
mv_status mv_token_logprob_bad_targets(const void* workspace, int32_t* host_count,
                                       hipStream_t stream);

/*
 * Gradient into the LM-head weights, dweight = G^T hidden (fp32 [vocab,
 * hidden]) with G_tv = dlogp_t (1[v = y_t] - softmax(z_t)_v), the same G that
 * mv_token_logprob_bwd writes into its workspace: call it with that workspace
 * after the backward, before the workspace is reused (the G it holds is not
 * validated).  n_tokens == 0 is a no-op (dweight is not written).
 */
mv_status mv_token_logprob_dweight(const mv_logprob_shape* shape, const void* hidden,
                                   const void* workspace, size_t workspace_bytes,
                                   float* dweight, hipStream_t stream);

/*
 * dlogp_t = d/dlogp_t [ -scale * min(ratio_t A_t, clamp(ratio_t) A_t) ]: the
 * clipped surrogate's gradient, zero where the clipped branch is active.
 */
mv_status mv_ppo_clip_dlogp(int32_t n, const float* ratio, const float* adv,
                            float eps_low, float eps_high, float scale,
                            float* dlogp, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * GRPO token loss and drift diagnostics (training recipe of Appendix F; the
 * ratio, advantage weight and KL term of a token all use its live-view
 * log-prob, Propositions "rl_tree" / "rl_4d"; drift is Eq. "logdiff").
 *
 * Trajectories are packed back to back: traj_ptr (device int32 [n_traj + 1])
 * holds their first token positions, traj_ptr[0] = 0 and traj_ptr[n_traj] =
 * n_tokens, non-decreasing (a malformed array gives unspecified results but
 * no access outside the arrays).  Consecutive runs of group_size trajectories
 * are the sample groups of one prompt.
 *
 *   A_i      = (r_i - mean_group r) / (std_group r + adv_eps)   (sample std,
 *              n - 1; 0 for a group of one)
 *   rho_t    = exp(logp_t - logp_old_t)          (logp_old: rollout log-prob)
 *   surr_t   = min(rho_t A, clamp(rho_t, 1 - eps_low, 1 + eps_high) A)
 *   k3_t     = exp(ref_t - logp_t) - (ref_t - logp_t) - 1   (reference KL)
 *   loss     = mean over loss tokens of (-surr_t + beta k3_t)
 *   dlogp_t  = d loss / d logp_t (0 off the loss mask), the upstream gradient
 *              of mv_token_logprob_bwd.
 * Inputs fp32 [n_tokens] (device); loss_mask uint8 [n_tokens] (null: every
 * token); logp_ref may be null only with beta == 0.  advantage (fp32
 * [n_traj], nullable) receives A.  stats (device) receives, in order: loss,
 * logdiff (mean |logp - logp_old| over loss tokens), the fractions of loss
 * tokens whose clipped term is active on the low and the high side, mean k3,
 * mean ratio, the number of loss tokens, mean |A| over trajectories.  Every
 * reduction runs in a fixed order (bitwise reproducible).
 * ------------------------------------------------------------------------ */
typedef struct {
  int32_t n_tokens, n_traj, group_size;
  float eps_low, eps_high;        /* clip pair, each in [0, 1)            */
  float beta;                     /* reference-KL weight (0: off)         */
  float adv_eps;                  /* added to the group std               */
} mv_grpo_shape;

typedef struct {
  float loss, logdiff, clip_frac_low, clip_frac_high, kl_ref, ratio_mean, n_loss_tokens,
      adv_abs_mean;
} mv_grpo_stats;

size_t mv_grpo_loss_workspace_bytes(const mv_grpo_shape* shape);

mv_status mv_grpo_loss(const mv_grpo_shape* shape, const int32_t* traj_ptr, const float* reward,
                       const float* logp, const float* logp_old, const float* logp_ref,
                       const uint8_t* loss_mask, float* advantage, float* dlogp,
                       mv_grpo_stats* stats, void* workspace, size_t workspace_bytes,
                       hipStream_t stream);

/*
 * mv_token_logprob and mv_grpo_loss in one forward: the GRPO loss terms, the
 * gradient dlogp and the drift statistics are evaluated in the log-prob's
 * combine pass, from its own logp, with no per-token array read back.
 * Outputs as the two calls give them (logp, ratio, clipped, lse as
 * mv_token_logprob with logp_old; advantage, dlogp, stats as mv_grpo_loss on
 * that logp): logp, ratio, clipped, lse, advantage and dlogp are bit-identical
 * to theirs; the statistics agree up to the order of their fp32 partial sums
 * (per 4 tokens here), fixed, so still bitwise reproducible.  dlogp is ready
 * for mv_token_logprob_bwd.  shape->eps_* clip the ratio output, grpo->eps_*
 * the loss (normally the same pair); grpo->n_tokens must equal
 * shape->n_tokens.  logp_old, logp, ratio, clipped, lse and dlogp are
 * required (n_tokens > 0); advantage and loss_mask may be null; logp_ref may
 * be null only with beta == 0.  A token on the loss mask whose target is -1
 * enters the loss with logp 0, as in the two-call form.  The workspace
 * (device, >= mv_token_logprob_grpo_workspace_bytes) also serves
 * mv_token_logprob_bad_targets.
 */
size_t mv_token_logprob_grpo_workspace_bytes(const mv_logprob_shape* shape,
                                             const mv_grpo_shape* grpo);

mv_status mv_token_logprob_grpo(const mv_logprob_shape* shape, const mv_grpo_shape* grpo,
                                const void* hidden, const void* weight, const int32_t* target,
                                const float* logp_old, const int32_t* traj_ptr,
                                const float* reward, const float* logp_ref,
                                const uint8_t* loss_mask, float* logp, float* ratio,
                                float* clipped, float* lse, float* advantage, float* dlogp,
                                mv_grpo_stats* stats, void* workspace, size_t workspace_bytes,
                                hipStream_t stream);

/* ---------------------------------------------------------------------------
 * SDCC junction KL (Section 5.1, Eq. "soft_loss"; forward KL, teacher first).
 *
 * At each diverging leaf p the teacher distribution p = softmax(W h_T[p]) (the
 * policy under the live prefix, stop-gradient) and the student distribution
 * q = softmax(W h_S[p]) (under the final-walk prefix) give
 *     KL_p = sum_v p_v (log p_v - log q_v),
 * computed by streaming vocabulary tiles through the same MFMA engine as the
 * log-prob, never storing logits.  Teacher and student hidden rows are read in
 * place through row indices (e.g. teacher_rows / student_rows of
 * mv_view_mask_leaves applied to the hidden states of a live-view and a
 * final-walk pass).  Layouts: hidden_* bf16 [n_rows_*, hidden]; rows int32
 * [n_leaves] (device); weight bf16 [vocab, hidden]; per-leaf fp32 [n_leaves].
 * A row index outside [0, n_rows_*) is read as an all-zero hidden state (the
 * kernels never read outside the matrices).  hidden % 64 == 0; n_leaves == 0
 * is a no-op.  The workspace (device, >= *_workspace_bytes, caller-owned) holds
 * per-leaf vocabulary-chunk partials (forward) or the bf16 rows dkl * (q - p)
 * (backward).
 * ------------------------------------------------------------------------ */
typedef struct {
  int32_t n_leaves, hidden, vocab;
  int32_t n_rows_teacher, n_rows_student;  /* rows of the two hidden matrices */
} mv_kl_shape;

size_t mv_sdcc_kl_workspace_bytes(const mv_kl_shape* shape);

mv_status mv_sdcc_kl(const mv_kl_shape* shape, const void* hidden_teacher,
                     const int32_t* teacher_rows, const void* hidden_student,
                     const int32_t* student_rows, const void* weight, float* kl,
                     float* lse_teacher, float* lse_student, void* workspace,
                     size_t workspace_bytes, hipStream_t stream);

size_t mv_sdcc_kl_bwd_workspace_bytes(const mv_kl_shape* shape);

/*
 * dh_student[p] = dkl[p] * (q - p)^T W  (bf16 [n_leaves, hidden]), the gradient
 * of sum_p dkl[p] KL_p into the student hidden state of each leaf (the teacher
 * is stop-gradient).  Logits are recomputed from the forward's LSEs.
 */
mv_status mv_sdcc_kl_bwd(const mv_kl_shape* shape, const void* hidden_teacher,
                         const int32_t* teacher_rows, const void* hidden_student,
                         const int32_t* student_rows, const void* weight,
                         const float* lse_teacher, const float* lse_student, const float* dkl,
                         void* dh_student, void* workspace, size_t workspace_bytes,
                         hipStream_t stream);

/*
 * The KL weight schedule of the training recipe (Appendix F): lambda ramps
 * linearly from 0 to lambda_max over the first warmup_frac of total_steps and
 * stays there.  Host only.
 */
float mv_sdcc_lambda(int32_t step, int32_t total_steps, float lambda_max, float warmup_frac);

/* ---------------------------------------------------------------------------
 * Kernel timing (measurement support, not part of the method).
 *
 * While enabled, every kernel the library enqueues is bracketed by a pair of
 * HIP events recorded on the launch stream.  mv_profile_enable(1) clears the
 * previous records; mv_profile_read waits for the recorded events and returns
 * the summed duration (ms) and launch count of the kernels named `kernel`
 * (one of "attn_fwd", "attn_bwd_dkdv", "attn_bwd_reduce",
 * "attn_bwd_dq", "lm_logits", "lm_combine", "lm_grad", "lm_dh", "lm_dw", "kl_logits",
 * "kl_combine", "kl_grad", "kl_dh", "grpo", "pack", "unpack", "rope", "materialize",
 * "ppo_clip").  Not for use
 * under stream capture.
 * ------------------------------------------------------------------------ */
mv_status mv_profile_enable(int32_t on);
mv_status mv_profile_read(const char* kernel, double* total_ms, int32_t* count);

#ifdef __cplusplus
}
#endif
#endif /* MV_H_ */
