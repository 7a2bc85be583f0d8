/*
 * la.h -- C ABI of libla: block selection and block-sparse attention for
 * autoregressive (AR) chunk generation on AMD Instinct MI355X (gfx950).
 *
 * The operation is the block-sparse attention of Light Interaction (Sec. 3.3): a chunk of Lq query tokens (the frames being
 * denoised) attends to Lk keys laid out as
 *     [n_text text tokens][historical visual context][current chunk: last Lq keys].
 * Tokens are cut into 1-D blocks of `block` consecutive tokens.  Per (batch, head,
 * query block i) the library
 *   1. pools each query block and each historical key block into its mean
 *      (Sec. 3.3, pooling equation);
 *   2. scores s_{i,m} = q_bar_i . k_bar_m / sqrt(d) over the M historical blocks
 *      (Sec. 3.3, selection equation);
 *   3. keeps a subset S_i of the historical blocks: either the shortest
 *      highest-scoring prefix whose softmax mass over the M scores reaches tau
 *      (la_select_blocks), or the floor(r*M) highest scores, the paper's own
 *      Top-floor(rM) rule (la_select_blocks_topk);
 *   4. attends over C_i = text blocks u current-chunk blocks u S_i (Sec. 3.3,
 *      context-union equation), the same block set for K and V.
 *
 * Conventions shared by every call
 *   - Tensors are device pointers, contiguous, row-major, layout [B, H, L, d]
 *     for q, k, v and o; bf16 is raw IEEE bfloat16 (16-bit), 16-byte aligned.
 *   - The caller owns every buffer.  The library allocates no memory and keeps
 *     no state between calls; scratch space comes in through `ws`/`ws_bytes`
 *     (size from la_workspace_bytes; 256-byte alignment).
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = default stream) and the
 *     call returns without synchronising.  Outputs are ready when the stream is.
 *   - Arguments are validated before anything is enqueued: on any error the call
 *     returns a non-zero la_status and enqueues nothing, writes nothing.
 *     LA_ERR_HIP reports a failed kernel launch (outputs are then undefined).
 *   - No floating-point atomics: results are bit-reproducible run to run.
 *   - Calls are thread-safe (no global state).
 *   - The selection and attention calls enqueue kernel launches only (no memset,
 *     copy, allocation or synchronisation), so a caller may capture them in a
 *     HIP graph; replays give the same results as the calls.  Exceptions:
 *     la_sparse_attn_schedule (a reading tool) enqueues copies, and the first
 *     la_select_blocks_noalloc call on a device looks up its scratch address
 *     (make that call before capturing).
 */
#ifndef LA_H_
#define LA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum la_status {
  LA_OK = 0,
  LA_ERR_ARG = 1,        /* null pointer, tau <= 0 or NaN, bad r, misaligned pointer */
  LA_ERR_SHAPE = 2,      /* unsupported or inconsistent shape (see la_shape) */
  LA_ERR_WORKSPACE = 3,  /* ws too small or NULL while needed */
  LA_ERR_HIP = 4         /* a HIP launch failed */
} la_status;

/* Problem shape.
 *   B, H        batch and heads (>= 1); every (b, h) is independent (Sec. 3.3:
 *               pooling and selection run per attention head).
 *   Lq, Lk      query tokens and key tokens, 1 <= Lq <= Lk - n_text.
 *   d           head dimension: 64 or 128.
 *   block       tokens per block, the same tiling for queries and keys: 64 or 128.
 *               NQ = ceil(Lq/block) query blocks, NK = ceil(Lk/block) key blocks.
 *   n_text      leading text-condition keys, always kept (the paper's T).
 *   frame_tokens  0: every kept key is visible to every query.  F > 0: frame-causal
 *               inside the chunk, query token t (chunk position) sees chunk key
 *               n (n >= Lk - Lq) only if (n - (Lk - Lq)) / F <= t / F; context keys
 *               stay visible.  Used by the attention calls only.
 * Key block m is forced (always kept, never scored) when it overlaps the text
 * tokens [0, n_text) or the chunk [Lk - Lq, Lk); the others are the M historical
 * candidates, block indices [ceil(n_text/block), floor((Lk-Lq)/block)).
 * Limits: NK <= 16384, M <= 4096, B*H <= 65535, and B*H*ceil(Lq/256)*NK*(block/64)
 * < 2^31 (the 64-key tiles of the attention work plan have 32-bit indices). */
typedef struct la_shape {
  int32_t B, H, Lq, Lk, d;
  int32_t block;
  int32_t n_text;
  int32_t frame_tokens;
} la_shape;

/* Bytes of scratch space the selection and attention calls need for this shape
 * (the maximum over them; the attention pass keeps its work plan and the partial
 * results of work split across workgroups there).  One ws may serve all calls in
 * stream order; a selection call overwrites an attention plan held in the same ws.
 * Returns 0 for an invalid shape. */
size_t la_workspace_bytes(const la_shape* shape);

/* Cumulative-mass block selection.
 *   q      bf16 [B, H, Lq, d];  k  bf16 [B, H, Lk, d]      (inputs)
 *   tau    in (0, +inf): per query block keep the shortest prefix of historical
 *          blocks, ordered by score descending (lower block index first on equal
 *          scores), whose softmax mass (softmax over the M scores) is >= tau.
 *          tau >= 1 keeps every historical block.
 *   mask   uint8 [B, H, NQ, NK] or NULL: 1 = key block kept, 0 = skipped.
 *   counts int32 [B, H, NQ]: number of kept key blocks per query block.
 *   idx    int32 [B, H, NQ, NK]: per query block, the kept key-block indices in
 *          ascending order in the first counts[] slots; later slots untouched.
 * Returns LA_ERR_ARG for tau <= 0 or NaN. */
la_status la_select_blocks(const la_shape* shape, const void* q, const void* k, float tau,
                           uint8_t* mask, int32_t* counts, int32_t* idx,
                           void* ws, size_t ws_bytes, void* stream);

/* la_select_blocks with no workspace argument, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  The scratch it needs (pooled queries and the score matrix,
 * la_workspace_bytes' selection part) is a device array of LA_NOALLOC_SCRATCH_BYTES
 * inside the library, one per GPU, held from the library's load until the process ends;
 * the call itself allocates nothing.
 *   Arguments, rule, outputs and errors as la_select_blocks; shapes whose selection
 *   scratch exceeds LA_NOALLOC_SCRATCH_BYTES (4 B * B*H*NQ*(d + M), rounded up to 256 B per
 *   part) return LA_ERR_WORKSPACE.  Every benchmark shape fits (at most 10.6 MB).
 *   The scratch belongs to the current device (hipGetDevice), which must be the device
 *   of q, k and the stream.  All calls on one GPU share it: calls that may overlap on one
 *   GPU (concurrent streams, or threads enqueueing at once) race; calls ordered on one
 *   stream do not.  Nothing carries over between calls (each call writes every scratch
 *   byte it reads). */
#define LA_NOALLOC_SCRATCH_BYTES (16u << 20)
la_status la_select_blocks_noalloc(const la_shape* shape, const void* q, const void* k, float tau,
                                   uint8_t* mask, int32_t* counts, int32_t* idx, void* stream);

/* The paper's Top-floor(rM) rule (Sec. 3.3, selection equation): keep the
 * keep_blocks = floor(r*M) highest-scoring historical blocks, computed by the
 * caller and clamped to [0, M] here (0 keeps only the forced blocks).  Same
 * outputs as la_select_blocks.  keep_blocks < 0 is LA_ERR_ARG. */
la_status la_select_blocks_topk(const la_shape* shape, const void* q, const void* k,
                                int32_t keep_blocks, uint8_t* mask, int32_t* counts,
                                int32_t* idx, void* ws, size_t ws_bytes, void* stream);

/* Block-sparse attention forward over the kept blocks.
 *   q bf16 [B, H, Lq, d]; k, v bf16 [B, H, Lk, d]                 (inputs)
 *   counts int32 [B, H, NQ], idx int32 [B, H, NQ, NK]: kept key blocks per query
 *          block in the first counts[] slots (as written by la_select_blocks or
 *          la_mask_to_list).  The set of listed blocks is used: order and repeats
 *          do not matter, entries outside [0, NK) are ignored and counts[] is
 *          clamped to [0, NK].  One list serves both K and V (Sec. 3.3).
 *   scale  logit scale; <= 0 selects 1/sqrt(d).
 *   o      bf16 [B, H, Lq, d]: o_t = sum_n softmax_n(q_t . k_n * scale) v_n over
 *          the keys of the kept blocks visible to t; 0 when none is.
 *   lse    float [B, H, Lq] or NULL: natural-log sum of exp(logits) per query
 *          token, -inf when no key is visible.
 * Softmax in fp32, products in bf16 with fp32 accumulation. */
la_status la_sparse_attn_fwd(const la_shape* shape, const void* q, const void* k, const void* v,
                             const int32_t* counts, const int32_t* idx, float scale,
                             void* o, float* lse, void* ws, size_t ws_bytes, void* stream);

/* la_sparse_attn_fwd in its three steps, for callers that time or reuse them.
 * The work plan depends only on the lists: units of 256 query rows (query blocks of a
 * head grouped by the first historical entry of their lists, the first kept historical
 * block for the ascending lists the selection writes; any order gives the same results),
 * the union of their lists as
 * 64-key tiles, and the split of the work over one persistent workgroup per CU of the
 * current device: whole units in rounds (the workgroups of one XCD start consecutive
 * units of a head together), the remaining and the longest units in equal-work shares
 * cut anywhere.  It lives in ws and is for the device it was built on.
 *
 * la_sparse_attn_plan: builds the plan for `shape` from counts/idx (read as in
 *   la_sparse_attn_fwd) into ws.
 * la_sparse_attn_run: the attention pass over the plan in ws (built by
 *   la_sparse_attn_plan for the same shape; it may be run for several q, k, v that
 *   share the lists).  Writes o and lse for the query rows of units processed whole by
 *   one workgroup, and partial results (O, running max, sum) into ws for the others.
 * la_sparse_attn_merge: merges those partials into o and lse (the buffers given to the
 *   run; lse may be NULL if it was NULL there).
 * Plan, run and merge must follow each other on one stream with the same ws, with no other
 * call using that ws in between (a selection call overwrites the plan): a run on a plan the
 * workspace no longer holds writes wrong values, though every access stays inside q, k, v, o,
 * lse and ws.  Arguments, alignment and errors as for la_sparse_attn_fwd. */
la_status la_sparse_attn_plan(const la_shape* shape, const int32_t* counts, const int32_t* idx,
                              void* ws, size_t ws_bytes, void* stream);
la_status la_sparse_attn_run(const la_shape* shape, const void* q, const void* k, const void* v,
                             float scale, void* o, float* lse, void* ws, size_t ws_bytes,
                             void* stream);
la_status la_sparse_attn_merge(const la_shape* shape, void* o, float* lse, void* ws,
                               size_t ws_bytes, void* stream);

/* The schedule of the plan in ws, for tools and tests that check or study it; it changes
 * nothing.  Units u < U = B H ceil(Lq / 256) own T tiles in all, ordered in one tile
 * sequence; the run's P persistent workgroups (one per CU of the current device, a multiple
 * of 8, at most 256) each take a range of whole units and a share cut anywhere.  Written:
 *   *P, *U    (host)  the two counts the arrays below are sized by;
 *   tstart    int32 [U + 1] (device): position of unit u's first tile; tstart[U] = T;
 *   ucount    int32 [U]     (device): 64-key tiles of unit u's list union (a unit with 0 still
 *             runs one tile, so it takes max(1, ucount[u]) positions);
 *   dp_start  int32 [P + 1] (device): workgroup l runs the whole units on [dp_start[l],
 *             dp_start[l + 1]) (rounds: its XCD's consecutive units);
 *   sk_start  int32 [P + 1] (device): and its share [sk_start[l], sk_start[l + 1]) of the
 *             remaining tiles, which starts at dp_start[P].
 * Any of the four arrays may be NULL (not copied); the copies run on `stream`.  The values
 * describe the plan la_sparse_attn_plan(_valid) built for `shape` on this device, as long as
 * no other call has used ws since; otherwise they are meaningless.  LA_ERR_ARG if P or U is
 * NULL; workspace errors as for la_sparse_attn_run. */
la_status la_sparse_attn_schedule(const la_shape* shape, const void* ws, size_t ws_bytes,
                                  int32_t* P, int32_t* U, int32_t* tstart, int32_t* ucount,
                                  int32_t* dp_start, int32_t* sk_start, void* stream);

/* Compacts a block mask (uint8 [B, H, NQ, NK], non-zero = kept) into the
 * counts/idx form la_sparse_attn_fwd reads.  Needs no workspace. */
la_status la_mask_to_list(const la_shape* shape, const uint8_t* mask, int32_t* counts,
                          int32_t* idx, void* stream);

/* ------------------------------------------------------------------------------
 * 3-D block layout (Sec. 3.3: visual tokens in non-overlapping (B_t, B_h, B_w)
 * blocks; the fused Q-Prep, KV-Prep and Untile Scatter of its operator fusion).
 *
 * Linear (AR) order: keys are [n_text text tokens][T_ctx context frames][T_q chunk
 * frames], queries are the T_q chunk frames; a frame is Hs x Ws tokens in raster
 * order, token (t, y, x) of a run of frames at (t Hs + y) Ws + x.
 * Blocks: the text in 1-D blocks of `block` tokens; each run of frames (context,
 * chunk) in 3-D blocks of bt x bh x bw tokens, in raster order of their block
 * coordinates, cut at the grid edges (fewer tokens there).  Inside a 3-D block,
 * tokens are in raster order.
 * Block-major (tiled) buffers give every block `block` slots: its tokens first, in
 * the order above, then zero padding.  Key blocks: NT = ceil(n_text/block) text
 * blocks, NC context blocks, NQ chunk blocks; query blocks: the NQ chunk blocks.
 * The tiled problem is the la_shape written by la_grid3d_shape (Lq = NQ block,
 * Lk = (NT + NC + NQ) block, n_text = NT block, frame_tokens = 0), so text and
 * chunk blocks are forced and the NC context blocks are the historical candidates.
 * The padding of key blocks is masked through the per-block valid counts
 * (la_grid3d_valid, la_sparse_attn_fwd_valid); padded query rows are dropped by
 * la_untile_o_3d.
 * -------------------------------------------------------------------------- */
typedef struct la_grid3d {
  int32_t B, H, d;       /* batch, heads, head dimension (64 or 128) */
  int32_t n_text;        /* text tokens (>= 0) */
  int32_t T_ctx, T_q;    /* context frames (>= 0) and chunk frames (>= 1) */
  int32_t Hs, Ws;        /* latent frame height and width in tokens (>= 1) */
  int32_t bt, bh, bw;    /* 3-D block extents (>= 1), bt*bh*bw <= block */
  int32_t block;         /* slots per block in the tiled buffers: 64 or 128 */
} la_grid3d;

/* Part bits of la_prep_kv_3d: which regions of the tiled K/V buffers to write. */
enum { LA_PART_TEXT = 1, LA_PART_CONTEXT = 2, LA_PART_CHUNK = 4, LA_PART_ALL = 7 };

/* Host-only.  Validates the grid and writes the la_shape of the tiled problem.
 * LA_ERR_ARG for NULL pointers, LA_ERR_SHAPE for an invalid grid or a tiled shape
 * la_shape does not accept. */
la_status la_grid3d_shape(const la_grid3d* grid, la_shape* tiled);

/* Host-only.  Valid tokens per block, into host arrays: qvalid int32 [NQ] (may be
 * NULL) and kvalid int32 [NT + NC + NQ] (may be NULL). */
la_status la_grid3d_valid(const la_grid3d* grid, int32_t* qvalid, int32_t* kvalid);

/* Fused Q-Prep (Sec. 3.3, operator fusion; pooling equation): one pass over the
 * chunk queries that writes them block-major and pools every query block.
 *   q        bf16 [B, H, T_q Hs Ws, d], linear order                    (input)
 *   q_tiled  bf16 [B, H, NQ block, d]: block-major, padding slots zero
 *   qbar     float [B, H, NQ, d] or NULL: mean of each block's tokens (fp32 sums) */
la_status la_prep_q_3d(const la_grid3d* grid, const void* q, void* q_tiled, float* qbar, void* stream);

/* Fused KV-Prep (Sec. 3.3, operator fusion; pooling equation): reads K and V
 * together, writes the regions named in `parts` of the block-major buffers and
 * pools the K blocks it writes.  Regions not named are left untouched (a text or
 * context region written once can be kept across calls).
 *   k, v      bf16 [B, H, n_text + (T_ctx + T_q) Hs Ws, d], linear order   (inputs)
 *   k_tiled, v_tiled  bf16 [B, H, (NT + NC + NQ) block, d]
 *   kbar      float [B, H, NT + NC + NQ, d] or NULL: block means of K (rows of the
 *             written regions only)
 *   parts     non-zero subset of LA_PART_ALL, else LA_ERR_ARG. */
la_status la_prep_kv_3d(const la_grid3d* grid, const void* k, const void* v, uint32_t parts,
                        void* k_tiled, void* v_tiled, float* kbar, void* stream);

/* Block means of a 1-D block layout (Sec. 3.3, pooling equation), for callers that keep the
 * key means of the context across calls (the context keys do not change between the
 * denoising steps of a chunk; the paper computes them once, when K enters its KV buffer) and
 * select with la_select_pooled.
 *   which  LA_POOL_Q: x = q bf16 [B, H, Lq, d] -> xbar float [B, H, NQ, d];
 *          LA_POOL_K: x = k bf16 [B, H, Lk, d] -> xbar float [B, H, NK, d].
 *   A ragged last block is the mean of its valid rows.  Sums in fp32, then one multiply by
 *   1 / rows: the same values la_select_blocks pools internally, so selecting from them with
 *   la_select_pooled gives la_select_blocks' result.
 * A bad `which`, NULL or misaligned pointers are LA_ERR_ARG.  Needs no workspace. */
enum { LA_POOL_Q = 0, LA_POOL_K = 1 };
la_status la_pool_blocks(const la_shape* shape, const void* x, int32_t which, float* xbar, void* stream);

/* Block selection from pooled means (Sec. 3.3, selection equation), for block
 * layouts pooled elsewhere (la_pool_blocks, la_prep_q_3d, la_prep_kv_3d).
 *   shape  the tiled shape; qbar float [B, H, NQ, d], kbar float [B, H, NK, d] (rows
 *          of the M historical blocks are read).
 * Rules, outputs and errors as la_select_blocks / la_select_blocks_topk. */
la_status la_select_pooled(const la_shape* shape, const float* qbar, const float* kbar, float tau,
                           uint8_t* mask, int32_t* counts, int32_t* idx, void* ws, size_t ws_bytes,
                           void* stream);
la_status la_select_pooled_topk(const la_shape* shape, const float* qbar, const float* kbar,
                                int32_t keep_blocks, uint8_t* mask, int32_t* counts, int32_t* idx,
                                void* ws, size_t ws_bytes, void* stream);

/* la_sparse_attn_fwd / la_sparse_attn_plan for key blocks with padding.
 *   kvalid  int32 [NK] device array: key block m holds valid keys at its first
 *           kvalid[m] slots (clamped to [0, block]); the others are invisible.
 *           NULL = every slot valid (the plain calls).
 * la_sparse_attn_run and la_sparse_attn_merge serve both plans unchanged. */
la_status la_sparse_attn_fwd_valid(const la_shape* shape, const void* q, const void* k, const void* v,
                                   const int32_t* counts, const int32_t* idx, const int32_t* kvalid,
                                   float scale, void* o, float* lse, void* ws, size_t ws_bytes,
                                   void* stream);
la_status la_sparse_attn_plan_valid(const la_shape* shape, const int32_t* counts, const int32_t* idx,
                                    const int32_t* kvalid, void* ws, size_t ws_bytes, void* stream);

/* Fused Untile Scatter (Sec. 3.3, operator fusion): block-major attention output back
 * to linear order; padding slots are dropped.
 *   o_tiled   bf16 [B, H, NQ block, d]; lse_tiled float [B, H, NQ block] or NULL (inputs)
 *   o         bf16 [B, H, T_q Hs Ws, d]; lse float [B, H, T_q Hs Ws] (written when both
 *             lse pointers are given) */
la_status la_untile_o_3d(const la_grid3d* grid, const void* o_tiled, const float* lse_tiled, void* o,
                         float* lse, void* stream);

/* ------------------------------------------------------------------------------
 * The scalar policy around the path: adaptive context management (Sec. 3.1) and the
 * denoising cache (Sec. 3.2).  Only the latent dynamics runs on the GPU; the other
 * calls are host-only scalar rules (no GPU, no stream), exact in double precision.
 * Camera-pose similarities are inputs: the paper instantiates them with an FOV
 * overlap measure it does not define.
 * -------------------------------------------------------------------------- */
typedef enum la_dtype { LA_DTYPE_F32 = 0, LA_DTYPE_BF16 = 1 } la_dtype;

/* Workspace bytes of la_latent_mse (fp64 partial sums; 256-byte aligned). */
#define LA_LATENT_MSE_WS_BYTES 8192

/* Latent dynamics D_t = MSE(z_{t-1}, z_{t-2}) (Sec. 3.1, latent-dynamics equation): the mean
 * over all n values of (z_a - z_b)^2.
 *   z_a, z_b  device arrays of n values of `dtype` (fp32 or bf16), 16-byte aligned; any
 *             layout, the same for both (the mean runs over every latent dimension).
 *   out       device double: D_t.  Squares are summed in fp32 within 16-byte chunks and in
 *             fp64 beyond; the order is fixed by n, so the result is bit-reproducible.
 *   ws        LA_LATENT_MSE_WS_BYTES of device scratch.
 * n < 1, a bad dtype, NULL or misaligned pointers are LA_ERR_ARG. */
la_status la_latent_mse(const void* z_a, const void* z_b, int64_t n, int32_t dtype, double* out,
                        void* ws, size_t ws_bytes, void* stream);

/* Host-only.  Moving average D_bar_t = alpha D_t + (1 - alpha) D_bar_{t-1} (Sec. 3.1,
 * smoothing equation); D_bar_prev NULL starts the average with D_t.  alpha in (0, 1],
 * D_t >= 0, else LA_ERR_ARG. */
la_status la_dynamics_ema(double D_t, const double* D_bar_prev, double alpha, double* D_bar);

/* Host-only.  Temporal window L_t = clip(floor(L_m kappa / (D_bar + kappa)), 1, L_m)
 * (Sec. 3.1, window equation).  kappa > 0, L_m >= 1, D_bar >= 0, else LA_ERR_ARG. */
la_status la_temporal_window(double D_bar, double kappa, int32_t L_m, int32_t* L_t);

/* Host-only.  Pose gate (Sec. 3.1 retrieved-memory gate, Sec. 3.2 reuse condition):
 * *revisiting = 1 when max_j similarities[j] >= tau_pose (keep the retrieved memory, allow
 * denoising reuse), 0 for pure exploration or n = 0 (discard the retrieved memory).
 * similarities: host array of n floats; NaN entries are LA_ERR_ARG. */
la_status la_pose_revisiting(const float* similarities, int32_t n, float tau_pose, int32_t* revisiting);

/* Host-only.  Denoising-cache schedule over K steps (Sec. 3.2, reuse equation): source[i] =
 * the step whose model output step i uses, i for an evaluated step and 0 for the reused
 * intermediate steps 1..K-2 when reuse != 0 and K > 2; the model is evaluated at steps i with
 * source[i] == i.  source: host array of K int32.  K < 1 is LA_ERR_ARG. */
la_status la_denoise_schedule(int32_t K, int32_t reuse, int32_t* source);

/* Static description of a status code. */
const char* la_status_string(la_status status);

/* ABI version of this header: 1. */
int32_t la_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LA_H_ */
