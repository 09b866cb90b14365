/*
 * hs.h — C ABI of libhs, the MI355X (gfx950) language-decode engine for
 * modality-disaggregated MLLM serving (arXiv 2603.12707).
 *
 * The boundary follows the paper's statement of the problem:
 *   - the payload that crosses the modality boundary is the projected visual
 *     embedding [1, N_v, d] (§5.1, §5.2 "Device Placement"), of N_v * d * b
 *     bytes (embedding-size display, §4.1);
 *   - the KV cache is allocated only when a request enters language prefill
 *     (§5.4 "Lazy KV Cache Allocation") and holds 2 * L * n_kv * d_h * s_ctx * b
 *     bytes per request (Eq. 1, §4.1), s_ctx = N_v + s_text (Theorem 1, §4.2);
 *   - N_v varies per request (§4.2 "Handling dynamic visual token counts",
 *     §5.2 "Aligned Batch Handoff");
 *   - decode is the memory-bandwidth-bound phase that streams the weights and
 *     the KV cache once per generated token (§2; Eq. 5, §4.3).
 *
 * Conventions
 *   - A KV handle serves any model created with the same hs_config whose
 *     max_ctx covers the handle's capacities (for instance copies of the
 *     weights); calls that take both reject any other (HS_E_INVALID).
 *   - Every call returns an int status: HS_OK (0) or a negative HS_E_* code;
 *     hs_last_error() returns a thread-local message for the last failure.
 *   - Device pointers are HIP device addresses on the device that was current
 *     when the model was created; they stay owned by the caller.  The library
 *     owns only what it allocates in hs_model_create / hs_kv_alloc
 *     (workspaces and per-request metadata) and frees it in the matching
 *     *_free call.
 *   - Calls taking a stream are asynchronous on that stream (NULL = the
 *     default stream).  hs_decode_step, hs_prefill_embeddings and
 *     hs_prefill_batch allocate no device memory and perform no
 *     device-to-host copy.
 *   - Argument, state and capacity checks run on host-side mirrors before any
 *     launch; a failing call launches nothing and changes no state.
 *
 * Storage dtype codes: HS_F32 (IEEE binary32), HS_F16 (binary16),
 * HS_BF16 (bfloat16).  Weights, vision rows, the KV cache and the
 * intermediate activations named below are stored in the model dtype; the
 * residual stream, logits and every accumulation are fp32; conversions to the
 * storage dtype round to nearest, ties to even.
 */
#ifndef HS_H
#define HS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HS_OK 0
#define HS_E_INVALID (-1)  /* NULL/negative/shape/dtype mismatch, n_v > capacity */
#define HS_E_CAPACITY (-2) /* a step would write position >= capacity */
#define HS_E_BUFFER (-3)   /* caller's KV buffer smaller than required */
#define HS_E_STATE (-4)    /* decode before prefill, prefill twice, ... */
#define HS_E_DEVICE (-5)   /* HIP runtime error (message in hs_last_error) */

#define HS_F32 0
#define HS_F16 1
#define HS_BF16 2

#define HS_ROPE_1D 0 /* rotate-half RoPE at the row's sequence position */
#define HS_ROPE_M3 1 /* 3-section multimodal RoPE driven by (t, h, w) ids */

typedef void *hs_stream_t; /* a hipStream_t */

/* Decoder shape.  d_model = any; head_dim even, head_dim / 2 a multiple of 16;
 * n_heads a multiple of n_kv_heads (query head i reads KV head
 * i / (n_heads / n_kv_heads)); d_model, n_heads * head_dim and ffn_dim
 * multiples of 8 (16-bit dtypes) or 4 (fp32).  For HS_ROPE_M3 the three
 * section sizes count frequency pairs and sum to head_dim / 2.  rope_theta and
 * rms_eps are used exactly as these fp32 values. */
typedef struct hs_config {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab;
  float rope_theta, rms_eps;
  int32_t rope_kind;
  int32_t mrope_section[3];
  int32_t qkv_bias;
  int32_t dtype;
} hs_config;

/* One decoder layer's weights, device pointers in the model dtype.  The
 * projection matrices are the nn.Linear matrices [out, in] in packed layout:
 *   wq [n_h*d_h, d]   wk, wv [n_kv*d_h, d]      written by hs_pack_matrix_heads
 *   wo [d, n_h*d_h]   w_gate, w_up [F, d]   w_down [d, F]   by hs_pack_matrix
 * the norm gains attn_norm, mlp_norm [d] and the optional biases
 * bq, bk, bv [rows] are plain vectors in the original row order. */
typedef struct hs_layer_weights {
  const void *attn_norm;
  const void *wq, *wk, *wv;
  const void *bq, *bk, *bv;
  const void *wo;
  const void *mlp_norm;
  const void *w_gate, *w_up;
  const void *w_down;
} hs_layer_weights;

/* embed [V, d] row-major (rows are gathered); final_norm [d]; lm_head [V, d]
 * packed by hs_pack_matrix.  lm_head == NULL declares a layer stack without a
 * head: decode then produces no tokens or logits. */
typedef struct hs_weights {
  const void *embed;
  const void *final_norm;
  const void *lm_head;
  const hs_layer_weights *layers; /* host array [n_layers] */
} hs_weights;

typedef struct hs_model hs_model;
typedef struct hs_kv hs_kv;

/* Thread-local description of the last failing call ("" if none). */
const char *hs_last_error(void);

/* KV-cache and embedding transfer sizes of one request (Eq. 1 and the
 * embedding-size display, §4.1):
 *   kv_bytes  = 2 * n_layers * n_kv_heads * head_dim * (n_v + s_text) * b
 *   emb_bytes = n_v * d_model * b
 * with b the dtype width; exact integers, no padding.  With
 * s_text = capacity - n_v it is also the size hs_kv_alloc lays out for one
 * request.  Pure host arithmetic; either output pointer may be NULL. */
int hs_kv_bytes(const hs_config *cfg, int64_t n_v, int64_t s_text, uint64_t *kv_bytes, uint64_t *emb_bytes);

/* Packed weight layout.  Decode streams every weight byte once per token, so
 * each projection matrix is stored in the order the GEMM reads it: the
 * row-major [rows, cols] matrix is cut into tiles of 16 rows; a tile is a
 * sequence of k-blocks of 256 bytes per row (128 elements for 16-bit dtypes,
 * 64 for fp32); k-block kb of tile t is four 1 KB sub-blocks s, and 16-byte
 * slot l = 16 * q + i of sub-block s holds the 16-byte chunk
 * c = 16 * kb + 4 * s + q of row 16 * t + i.  Rows past `rows` and chunks past
 * `cols` are zero.  cols must be a multiple of 8 (16-bit) or 4 (fp32).
 * hs_packed_bytes gives the size; hs_pack_matrix converts src (row-major,
 * device) into dst (device, hs_packed_bytes long, 16-byte aligned),
 * asynchronously on the stream. */
int hs_packed_bytes(int32_t dtype, int64_t rows, int64_t cols, uint64_t *bytes);
int hs_pack_matrix(int32_t dtype, const void *src, int64_t rows, int64_t cols, void *dst, hs_stream_t stream);

/* The packed layout of a q, k or v projection, whose rows form heads of
 * head_dim rows: as hs_pack_matrix after reordering every head's rows so that
 * row 2 j of the head is its row j and row 2 j + 1 its row j + head_dim / 2
 * (the pair that rotate-half RoPE turns together, so that one 16-row tile
 * holds whole pairs).  Same size as hs_packed_bytes;
 * head_dim must be a positive multiple of 16 that divides rows. */
int hs_pack_matrix_heads(int32_t dtype, const void *src, int64_t rows, int64_t cols, int32_t head_dim, void *dst,
                         hs_stream_t stream);

/* Validates cfg, records the caller-owned weight pointers (they must outlive
 * the model) and allocates the workspaces for decode batches of up to
 * max_batch requests and requests of up to max_ctx positions (prefill rows,
 * capacities and RoPE position ids are all < max_ctx).  Uses the current
 * HIP device. */
int hs_model_create(const hs_config *cfg, const hs_weights *w, int32_t max_batch, int32_t max_ctx, hs_model **out);
int hs_model_free(hs_model *m);

/* The per-request KV cache, taken when a request enters language prefill
 * (§5.4 "Lazy KV Cache Allocation") and sized by Eq. 1 (§4.1): request b
 * holds 2 * n_layers * n_kv * head_dim * capacity_b elements.
 * Lays out `batch` requests back to back, in order and without padding, in
 * the caller-owned device buffer dev_buf, which must hold at least
 * sum_b kv_bytes(capacity_b) bytes.  Request b occupies capacity[b]
 * positions; its KV element (layer l, K|V = s, kv head j, position p,
 * channel e) sits at element offset
 *   base_b + (((l * 2 + s) * n_kv + j) * capacity_b + p) * head_dim + e,
 *   base_b = sum_{b' < b} 2 * n_layers * n_kv * head_dim * capacity_b',
 * so that each (request, layer, K|V, head) is one contiguous
 * [capacity_b, head_dim] slab streamed row by row.  n_v[b] (host) is the
 * request's vision-row count, checked again at prefill; capacity[b] (host)
 * must satisfy 0 <= n_v[b] <= capacity[b] <= max_ctx.  All lengths start at 0.
 * The handle owns small device metadata arrays; dev_buf stays the caller's. */
int hs_kv_alloc(hs_model *m, int32_t batch, const int32_t *n_v, const int32_t *capacity, void *dev_buf,
                uint64_t buf_bytes, hs_kv **out);
int hs_kv_free(hs_kv *kv);

/* A block-granular KV cache for serving (§5.4 "Lazy KV Cache Allocation":
 * KV memory is taken only when a request enters prefill, and grows with it).
 * dev_buf (caller-owned, 16-byte aligned) is cut into blocks of block_tokens
 * positions; a block holds those positions for every (layer, K|V, KV head):
 * kv_bytes(block_tokens) = 2 * n_layers * n_kv * head_dim * block_tokens * b
 * bytes, and the buffer holds floor(buf_bytes / that) blocks.  Element
 * (layer l, K|V = s, kv head j, position p, channel e) of the request in
 * slot r sits at
 *   start(r, p / block_tokens) + (((l * 2 + s) * n_kv + j) * block_tokens
 *                                 + p % block_tokens) * head_dim + e,
 * start(r, k) being the element offset of the k-th block the slot holds.
 * The handle has `slots` slots (1..4096), all empty; block_tokens is a power
 * of two in 256..16384 (decode attention reads a block in whole batches of
 * up to 256 positions); 16-bit storage only.  Blocks are handed out on the device, from a free list, as a slot's
 * length reaches them: at prefill for the context, and inside
 * hs_decode_step when a request enters a new block, so decode stays
 * graph-replayable.  hs_prefill_embeddings / hs_prefill_batch take slot
 * numbers as request numbers.  hs_decode_step runs over the slots holding a
 * prefilled request, in slot order; tokens_in / tokens_out are indexed by
 * slot ([slots]; other entries untouched) and logits / hidden_out rows
 * follow that order.  Host-side checks refuse a prefill or step the free
 * blocks cannot cover (HS_E_CAPACITY) before launching anything. */
int hs_kv_pool_create(hs_model *m, int32_t slots, int32_t block_tokens, void *dev_buf, uint64_t buf_bytes,
                      hs_kv **out);
/* Puts a request (n_v vision rows, at most `capacity` positions,
 * capacity <= max_ctx) in an empty slot of a pooled cache; takes no block. */
int hs_kv_admit(hs_kv *kv, int32_t slot, int32_t n_v, int32_t capacity, hs_stream_t stream);
/* Ends the slot's request: its blocks return to the free list and the slot
 * is empty again.  Stream-ordered: work queued before it on `stream` still
 * sees the blocks. */
int hs_kv_release(hs_kv *kv, int32_t slot, hs_stream_t stream);
/* Measurement: reads `bytes` (a positive multiple of 16) of device memory at
 * buf (16-byte aligned) with the same 16-byte non-temporal loads the kernels
 * stream weights with, each work group 32 KB of consecutive bytes at a time,
 * writing one word per work group to sink (device, [blocks]) so the reads
 * cannot be skipped.  The plain HBM read rate that the kernels' own rates are
 * compared with. */
int hs_stream_read(const void *buf, uint64_t bytes, uint32_t *sink, int32_t blocks, hs_stream_t stream);

/* Aligned batch handoff (§5.2 "Aligned Batch Handoff"): requests whose
 * projected embeddings have arrived wait in arrival order until a batch for
 * hs_prefill_batch is due.  A batch is the longest arrival-order prefix of
 * at most `align` requests (the paper's B_align, 32 by default) whose rows
 * fit max_rows (0: no budget; one request always fits).  It is due when it
 * holds `align` requests, when the row budget closes it with more requests
 * waiting, or when its oldest request has waited timeout_ms (the paper's
 * 500 ms) -- so an under-filled batch still goes.  Times are the caller's
 * clock in milliseconds, non-decreasing across pushes.  Host only; not
 * thread-safe.  max_pending (>= align) bounds the queue: a push beyond it
 * fails with HS_E_CAPACITY. */
typedef struct hs_handoff hs_handoff;
int hs_handoff_create(int32_t align, int64_t max_rows, int32_t max_pending, double timeout_ms, hs_handoff **out);
int hs_handoff_free(hs_handoff *h);
/* request `req` (>= 0), with `rows` context rows to prefill, arrived at now_ms */
int hs_handoff_push(hs_handoff *h, int32_t req, int32_t rows, double now_ms);
/* If a batch is due at now_ms, moves its requests (in arrival order) to
 * reqs[0 .. *n) (room for max; HS_E_BUFFER if too small) and their row sum
 * to *rows; else *n = 0.  *wait_ms (may be NULL) gets the time until the
 * oldest waiting request times out (0 when due again at once, -1 when none
 * waits). */
int hs_handoff_pop(hs_handoff *h, double now_ms, int32_t *reqs, int32_t max, int32_t *n, int64_t *rows,
                   double *wait_ms);
int hs_handoff_pending(const hs_handoff *h, int32_t *n);

/* Free and total blocks of a pooled cache (host mirror; exact after
 * hs_kv_sync when graph replays have taken blocks). */
int hs_kv_pool_blocks(const hs_kv *kv, int32_t *free_blocks, int32_t *n_blocks);

/* Language prefill of request `req` from its projected visual embedding, the
 * payload that crosses the modality boundary (§5.1: the embedding [1, N_v, d]
 * enters the language model; §5.2 "Device Placement": the embedding is put
 * in the language GPU's HBM just before prefill starts, so this call takes
 * it as device memory):
 * rows 0..n_v-1 are emb [n_v, d] (device, model dtype), rows n_v..n_v+s_text-1
 * are the embeddings of text_ids [s_text] (device int32, 0 <= id < vocab).
 * RoPE: HS_ROPE_1D uses position r for row r and pos_thw must be NULL;
 * HS_ROPE_M3 needs pos_thw (device int32 [3][n_v + s_text], the (t, h, w) ids
 * of every row, each < max_ctx) and the next decode position becomes
 * max(pos_thw) + 1.  Fills KV positions [0, s_ctx), sets the request length to
 * s_ctx, writes the first generated token to first_token (device int32[1])
 * and, if last_logits is not NULL, the fp32 logits of the last row
 * (device [vocab]).  Requires the model to have an LM head and the request to
 * be empty (HS_E_STATE otherwise). */
int hs_prefill_embeddings(hs_model *m, hs_kv *kv, int32_t req, const void *emb, const int32_t *text_ids,
                          int32_t s_text, const int32_t *pos_thw, float *last_logits, int32_t *first_token,
                          hs_stream_t stream);

/* Language prefill of n requests at once (§5.4: prefill of the requests whose
 * embeddings have arrived; §5.2 "Aligned Batch Handoff" hands them over in
 * batches).  Their rows are packed request by request, each request's rows
 * as in hs_prefill_embeddings (vision rows, then text rows):
 *   reqs      host int32 [n], distinct requests of the handle, all empty;
 *   emb       device, model dtype: the vision rows of reqs[0], then of
 *             reqs[1], ... ([sum_i n_v(reqs[i])][d], n_v as given to
 *             hs_kv_alloc; 16-byte aligned; NULL if that sum is 0);
 *   text_ids  device int32: the text ids of reqs[0], then of reqs[1], ...
 *             ([sum_i s_text[i]]; NULL if that sum is 0);
 *   s_text    host int32 [n];
 *   pos_thw   HS_ROPE_M3: device int32 [3][R], R = sum_i (n_v + s_text[i]),
 *             section-major (all rows' t ids, then h, then w), rows packed as
 *             above; HS_ROPE_1D: NULL (row r of a request is position r);
 *   first_tokens  device int32 [n]: the first generated token of reqs[i];
 *   last_logits   device fp32 [n][vocab] or NULL.
 * The requests are taken in order, in passes of at most 32 requests whose rows
 * fit the model's row workspaces (max(max_batch, max_ctx) rows, or what
 * hs_model_reserve_rows set); with last_logits NULL a pass also holds at most
 * max_batch requests.  Each pass runs every layer once over all its rows:
 * the projections as GEMMs over the packed rows, attention causal within
 * each request.  Every check (requests, lengths, capacities, pointers) runs
 * before the first launch. */
int hs_prefill_batch(hs_model *m, hs_kv *kv, int32_t n, const int32_t *reqs, const void *emb,
                     const int32_t *text_ids, const int32_t *s_text, const int32_t *pos_thw, float *last_logits,
                     int32_t *first_tokens, hs_stream_t stream);

/* Grows the model's row workspaces (residual stream, q, attention and SwiGLU
 * outputs, normalised rows) to hold `rows` packed prefill rows, so that
 * hs_prefill_batch packs more requests per pass; never shrinks them.  It
 * allocates, and waits for the device to go idle before freeing the old
 * buffers: call it outside any stream capture and not from a serving loop.
 * When it grows them, a HIP graph captured earlier from this model's decode
 * steps still holds the freed buffers' addresses: capture it again before
 * replaying. */
int hs_model_reserve_rows(hs_model *m, int64_t rows);

/* One greedy decode step for every request of the handle: request b embeds
 * tokens_in[b] (device int32 [batch]), writes its K/V rows at position len_b,
 * attends over positions [0, len_b], and (with an LM head) writes the argmax
 * of its logits, lowest index on ties, to tokens_out[b] (device int32
 * [batch]; may not alias tokens_in).  The lengths advance on the device, so
 * repeated calls need no host input.  logits (device fp32 [batch, vocab]) and
 * hidden_out (device fp32 [batch, d], the residual stream after the last
 * layer) are optional outputs.  Errors: HS_E_STATE if a request is not
 * prefilled, HS_E_CAPACITY if len_b == capacity_b for some b.  Token ids
 * outside [0, vocab) are replaced by 0 and flagged (hs_model_status).
 * The call only enqueues kernels (and, with hidden_out, one device copy) on
 * the stream, with a launch configuration fixed by the handle, so it can be
 * recorded into a HIP graph (stream capture) and the graph replayed, one step
 * per replay, for as long as every request has capacity left: the checks
 * above run on host mirrors when the call is made, not at replay (the paper
 * captures its decode iteration with CUDA Graphs, §5.4).  After replays,
 * hs_kv_sync brings the host mirrors up to date. */
int hs_decode_step(hs_model *m, hs_kv *kv, const int32_t *tokens_in, int32_t *tokens_out, float *logits,
                   float *hidden_out, hs_stream_t stream);

/* hs_decode_step for callers that cannot allocate device memory (code under
 * stream capture, tight serving loops, harnesses that forbid hipMalloc): the
 * step's scratch -- residual stream, q / attention / SwiGLU / normalised-row
 * activations, K-split and attention-split partials, and the logits when
 * `logits` is NULL -- lives in one static device array of
 * HS_STATIC_SCRATCH_BYTES per GPU, held from the first call on that GPU
 * until the process ends, instead of the model's workspaces.  Arguments,
 * checks and results are those of hs_decode_step (the same kernels).  The
 * call allocates nothing; a step whose scratch would exceed the array (for
 * instance batch * vocab fp32 logits with logits NULL) fails with
 * HS_E_INVALID before any launch.  Every call on a GPU shares that GPU's
 * array: calls that overlap on one GPU (several streams, several host
 * threads) race, and the array keeps the last call's contents.  The
 * current device must be the model's. */
#define HS_STATIC_SCRATCH_BYTES (64ull << 20)
int hs_decode_step_static(hs_model *m, hs_kv *kv, const int32_t *tokens_in, int32_t *tokens_out, float *logits,
                          float *hidden_out, hs_stream_t stream);

/* Reads and clears the device-side flags.  Synchronises the device.
 *   bit 0 (1): a token id outside [0, vocab) was replaced by 0;
 *   bit 2 (4): a pooled cache ran out of free blocks inside a replayed decode
 *              step (the host-side check covers eager calls only).  The
 *              requests left without a block for their new position keep it
 *              unstored, attention masks that position, and their outputs
 *              from that step on are not the model's: release requests or
 *              give the pool room before replaying again. */
int hs_model_status(hs_model *m, int32_t *flags);

/* ---- kernel replay (measurement hook) ---- */

/* Kernel kinds of one decode step, in launch order within a layer. */
#define HS_K_EMBED 0   /* token embedding gather */
#define HS_K_QKV 1     /* RMSNorm + q/k/v projection + RoPE + KV append */
#define HS_K_ATTN 2    /* split-K attention over the KV cache */
#define HS_K_COMBINE 3 /* combine of the attention splits */
#define HS_K_OPROJ 4   /* output projection + residual */
#define HS_K_GATEUP 5  /* RMSNorm + gate/up projection + SwiGLU */
#define HS_K_DOWN 6    /* down projection + residual */
#define HS_K_HEAD 7    /* final RMSNorm + LM head */
#define HS_K_ARGMAX 8  /* greedy selection and length advance */
#define HS_K_COUNT 9

/* Launches `count` kernels of one kind back to back on the stream, in the
 * launch configuration of this handle's decode step, cycling over the layers
 * (layer i % n_layers), so that a caller can time one kernel with events
 * around the batch.  Only for measurement between decode steps: the replayed
 * kernels read and rewrite the step's workspaces (and q/k/v rewrites the
 * K/V rows at each request's next position, which the next step rewrites
 * again); lengths do not change.  Kinds: HS_K_QKV, HS_K_ATTN, HS_K_COMBINE
 * (HS_E_STATE when the batch runs attention in one split), HS_K_OPROJ,
 * HS_K_GATEUP, HS_K_DOWN, HS_K_HEAD.  Same state checks as hs_decode_step. */
int hs_replay_kernels(hs_model *m, hs_kv *kv, int32_t kind, int32_t count, hs_stream_t stream);

/* ---- test and fill hooks (synchronous) ---- */

/* Host copy of every request's current length (int32 [batch]). */
int hs_kv_lengths(const hs_kv *kv, int32_t *host_len);

/* Waits for the device and copies the lengths and RoPE positions into the
 * handle's host mirrors (needed after replaying a captured decode step, whose
 * advances happen on the device only). */
int hs_kv_sync(hs_kv *kv);

/* Copies n rows of head_dim elements (model dtype) into / out of the cache at
 * (req, layer, kv_sel 0 = K / 1 = V, head, positions pos0..pos0+n-1);
 * src_is_device selects whether src/dst is a device or a host pointer. */
int hs_kv_write(hs_kv *kv, int32_t req, int32_t layer, int32_t kv_sel, int32_t head, int32_t pos0, int32_t n,
                const void *src, int32_t src_is_device);
int hs_kv_read(const hs_kv *kv, int32_t req, int32_t layer, int32_t kv_sel, int32_t head, int32_t pos0, int32_t n,
               void *dst, int32_t dst_is_device);

/* Marks request req as holding `len` valid positions (filled through
 * hs_kv_write) with next RoPE position rope_pos, as a prefill would. */
int hs_kv_set_length(hs_kv *kv, int32_t req, int32_t len, int32_t rope_pos);

#ifdef __cplusplus
}
#endif
#endif
