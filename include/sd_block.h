/*
 * sd_block.h -- C ABI of libsdblock.so: the per-step hot path of diffusion-based
 * speculative decoding with instance-adaptive block sizes (BlockPilot,
 * arXiv 2606.31315), as hand-written HIP kernels for AMD MI355X (gfx950).
 *
 * One speculative step drafts a block of B tokens in one block-diffusion forward
 * pass and the target model verifies the whole block in one parallel forward pass,
 * accepting the longest consistent prefix (Sec. 2.1; Fig. 1 caption; App. A.1).
 * The block size is chosen once per prompt and then fixed (Sec. 2.4, Eq. 9), so a
 * batch carries ragged per-sequence block lengths B_s.  This library provides the
 * two data-parallel operations of that step:
 *
 *   sd_block_attn  block attention of the B_s block rows of every sequence over its
 *                  GQA key/value cache, causal inside the block (target verify) or
 *                  bidirectional inside the block (block-diffusion drafter);
 *   sd_accept      vocabulary-wide speculative acceptance: greedy matching at T = 0,
 *                  lossless rejection sampling against min(1, p/q) at T > 0, giving
 *                  the accepted prefix length and the bonus or resampled token.
 *
 * Conventions shared by every entry point
 *   - All array arguments are DEVICE pointers unless stated otherwise; shape
 *     structs are host pointers.  The caller owns every buffer; the library never
 *     allocates, frees or retains device memory, and keeps no mutable global state
 *     except a thread-local error message.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream of the
 *     current device).  Calls enqueue work and return; they never synchronise.
 *   - Every call validates its host-side arguments before touching the device and
 *     returns a status code; it never aborts or prints.  Per-sequence values that
 *     live in device memory (ctx_lens, block_lens, q_offsets, tokens) cannot be
 *     checked on the host: values outside the documented ranges are undefined
 *     behaviour (sd_check_attn_inputs and sd_check_accept_inputs test them on the device).
 *   - Workspace: each operation needs device scratch memory of the size its
 *     *_workspace_size() reports (partial results between the kernels of one
 *     call).  Its contents on entry do not matter.  Calls that share a workspace
 *     must not overlap in time (use one stream, or one workspace per stream).
 *   - Row-major layouts throughout; "[a, b, c]" lists dimensions outermost first.
 */
#ifndef SD_BLOCK_H
#define SD_BLOCK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes -------------------------------------------------------- */
enum {
  SD_OK = 0,
  SD_ERR_INVALID_ARG = 1, /* null pointer, bad size, misalignment, bad enum */
  SD_ERR_UNSUPPORTED = 2, /* valid request this build has no kernel for (head_dim, group size) */
  SD_ERR_WORKSPACE = 3,   /* workspace smaller than *_workspace_size() */
  SD_ERR_HIP = 4          /* a HIP runtime call or kernel launch failed */
};

/* ---- element types and masks --------------------------------------------- */
enum { SD_F32 = 0, SD_BF16 = 1 };

enum {
  /* Target verification: block row i of sequence s sees keys [0, ctx_s + i]. */
  SD_MASK_CAUSAL_IN_BLOCK = 0,
  /* Block-diffusion drafting: every block row of s sees keys [0, ctx_s + B_s). */
  SD_MASK_BIDIR_IN_BLOCK = 1
};

/* Thread-local message describing the last non-OK status of this thread. */
const char *sd_last_error(void);

/* Library version string, e.g. "sdblock 0.1 gfx950". */
const char *sd_version(void);

/* ==========================================================================
 * Block attention (Sec. 2.1: the drafter generates the B block tokens in parallel
 * by block-level diffusion; the target verifies the block in parallel).
 * ========================================================================== */
typedef struct sd_attn_shape {
  int32_t num_seqs;     /* S >= 0 */
  int32_t num_q_heads;  /* Hq >= 1 */
  int32_t num_kv_heads; /* Hkv >= 1, Hq % Hkv == 0; query head h reads kv head h / (Hq/Hkv) */
  int32_t head_dim;     /* D: 64 or 128 */
  int32_t max_kv_len;   /* Lmax: cache rows per (sequence, kv head) */
  int32_t total_q;      /* sum_s B_s: rows of q and out */
  int32_t max_ctx;      /* host-known bound: ctx_lens[s] <= max_ctx for every s */
  int32_t max_block;    /* host-known bound: block_lens[s] <= max_block, 1 <= max_block <= 64 */
  int32_t dtype;        /* SD_BF16 or SD_F32: element type of q, caches and out */
  float scale;          /* softmax scale; 0 means 1/sqrt(D) */
} sd_attn_shape;

/* Workspace bytes sd_block_attn needs for this shape (host-only, no device access). */
int sd_block_attn_workspace_size(const sd_attn_shape *shape, size_t *bytes);

/*
 * out[q_offsets[s] + i, h, :] = sum_j softmax_j(scale * q_i,h . K[s, g, j, :]) V[s, g, j, :]
 * with g = h / (Hq/Hkv) and j ranging over the keys the mask lets block row i see
 * (causal: j <= ctx_s + i; bidirectional: j < ctx_s + B_s).  Softmax and all sums
 * are computed in fp32; for bf16 the attention weights are rounded to bf16 before
 * they multiply V (the output is then rounded to bf16).
 *
 *   q, out          [total_q, Hq, D]           dtype; row q_offsets[s] + i is block position i of s
 *   k_cache,v_cache [S, Hkv, Lmax, D]          dtype; the block's own keys/values must already be
 *                                              written at rows [ctx_s, ctx_s + B_s); rows at or beyond
 *                                              ctx_s + B_s are never read
 *   ctx_lens        [S] int32                  committed context length ctx_s, 0 <= ctx_s <= max_ctx
 *   block_lens      [S] int32                  block length B_s, 0 <= B_s <= max_block (0: no rows)
 *   q_offsets       [S + 1] int32              exclusive prefix sum of block_lens, q_offsets[S] = total_q
 *   mask_mode       SD_MASK_*
 *   workspace       >= sd_block_attn_workspace_size() bytes, 256-byte aligned
 *
 * Host-checked preconditions: q, caches and out 16-byte aligned; max_ctx + max_block
 * <= Lmax; total_q <= S * max_block; (Hq/Hkv) * max_block <= 256.
 * Errors: SD_ERR_INVALID_ARG, SD_ERR_UNSUPPORTED (head_dim), SD_ERR_WORKSPACE, SD_ERR_HIP.
 * S == 0 or total_q == 0 returns SD_OK without touching the device.
 */
int sd_block_attn(const sd_attn_shape *shape, const void *q, const void *k_cache, const void *v_cache,
                  const int32_t *ctx_lens, const int32_t *block_lens, const int32_t *q_offsets,
                  int32_t mask_mode, void *out, void *workspace, size_t workspace_bytes, void *stream);

/*
 * Paged variant: the caches are pools of fixed-size pages shared by all sequences, as a
 * serving engine keeps them.  Logical key j of sequence s lives in pool page
 * block_table[s * max_pages + j / page_size] at row j % page_size:
 *   k_pages, v_pages [num_pages, Hkv, page_size, D] bf16
 *   block_table      [S, max_pages] int32 (device)
 * Everything else, including the result, is as in sd_block_attn (same workspace size);
 * shape->max_kv_len must equal max_pages * page_size.  page_size is a power of two in
 * [16, 4096].  Page ids outside [0, num_pages) are clamped into the pool (the result is then
 * meaningless, but no read leaves the pool).  bf16 only (SD_ERR_UNSUPPORTED otherwise).
 */
int sd_block_attn_paged(const sd_attn_shape *shape, int32_t page_size, int32_t num_pages, int32_t max_pages,
                        const int32_t *block_table, const void *q, const void *k_pages, const void *v_pages,
                        const int32_t *ctx_lens, const int32_t *block_lens, const int32_t *q_offsets,
                        int32_t mask_mode, void *out, void *workspace, size_t workspace_bytes, void *stream);

/*
 * sd_block_attn with the block's keys and values taken from the new rows rather than the
 * cache, and written into the cache by the same launch (the append before verification,
 * Sec. 2.1, fused into it):
 *   k_new, v_new    [total_q, Hkv, D] bf16: row q_offsets[s] + i is block position i of s
 *   k_cache,v_cache [S, Hkv, Lmax, D] bf16: rows [0, ctx_s) are read; rows [ctx_s, ctx_s + B_s)
 *                                     are written with the new rows (their old contents are
 *                                     never read)
 * The result equals sd_kv_append followed by sd_block_attn, bit for bit.  Everything else is
 * as in sd_block_attn (same workspace size).  bf16 only (SD_ERR_UNSUPPORTED otherwise).
 */
int sd_block_attn_append(const sd_attn_shape *shape, const void *q, const void *k_new, const void *v_new,
                         void *k_cache, void *v_cache, const int32_t *ctx_lens, const int32_t *block_lens,
                         const int32_t *q_offsets, int32_t mask_mode, void *out, void *workspace,
                         size_t workspace_bytes, void *stream);

/* ==========================================================================
 * Speculative acceptance (Fig. 1 caption: accept the longest consistent prefix;
 * Sec. 1 and Sec. 3.1: the target's output distribution is preserved exactly).
 * Block layout: position 0 of a block is the last committed token (the anchor),
 * positions 1 .. B_s-1 are drafted; so each sequence has B_s target rows,
 * B_s - 1 draft rows, accept_len in [0, B_s - 1] and one bonus/resampled token.
 * ========================================================================== */
typedef struct sd_accept_shape {
  int32_t num_seqs;  /* S >= 0 */
  int32_t vocab;     /* 1 <= V <= 2^28 */
  int32_t total_q;   /* sum_s B_s */
  int32_t max_block; /* host-known bound on B_s, 1 <= max_block <= 64 */
  int32_t dtype;     /* SD_BF16 or SD_F32: element type of both logit arrays */
} sd_accept_shape;

/* Workspace bytes sd_accept needs for this shape at this temperature (host-only): enough for
 * the tagged-word paths described under sd_accept where the shape allows them. */
int sd_accept_workspace_size(const sd_accept_shape *shape, float temperature, size_t *bytes);

/*
 *   target_logits [total_q, V]       row q_offsets[s] + i: target logits after block position i
 *   draft_logits  [total_q - S, V]   row q_offsets[s] - s + j: drafter logits for block position
 *                                    j + 1, j < B_s - 1 (read only when temperature > 0; may be NULL
 *                                    at temperature 0, or when every block holds only its anchor,
 *                                    total_q = S)
 *   draft_tokens  [total_q - S] int32  drafted token of block position j + 1, in [0, V) (a token
 *                                    outside that range is never accepted)
 *   uniforms      [total_q] fp32 in [0, 1): slot q_offsets[s] + j drives acceptance test j;
 *                                    slot q_offsets[s] + B_s - 1 drives the single final draw
 *                                    (read only when temperature > 0; may be NULL at 0)
 *   block_lens    [S] int32          1 <= B_s <= max_block (every block holds at least its anchor)
 *   q_offsets     [S + 1] int32      exclusive prefix sum of block_lens
 *   temperature   0: greedy (draft j accepted iff it equals the lowest-index argmax of target
 *                 row j; next token = argmax of target row accept_len).
 *                 > 0: p = softmax(target/T), q = softmax(draft/T); draft j accepted iff
 *                 u_j < p_j(d_j) / q_j(d_j); on the first rejection at j the next token is the
 *                 inverse-CDF draw (ascending vocabulary order, first token whose cumulative mass
 *                 exceeds u* times the total) from max(0, p_j - q_j), or from p_j if that
 *                 residual has no mass; with every draft accepted it is the draw from p_{B_s-1}.
 *   accept_len    [S] int32 out      number of leading accepted drafts
 *   next_token    [S] int32 out      bonus or resampled token
 *
 * Host-checked preconditions: logits 16-byte aligned; temperature finite and >= 0;
 * S <= total_q <= S * max_block; vocab <= 2^28.  Softmax statistics and per-chunk masses are
 * accumulated in fp32, the acceptance ratio and the final draw's cumulative sums in fp64;
 * decisions within about 1e-6 of a boundary may differ from an fp64 evaluation.
 *
 * Paths.  Where the workspace holds sd_accept_workspace_size bytes, the stream is not
 * capturing a graph and the shape allows it, workgroups hand partial results on through
 * tagged words in the workspace instead of kernel boundaries:
 *   T = 0: one launch (at most 8 statistics chunks of 32768 bf16 / 16384 fp32 logits per row,
 *          at most 1024 sequences) instead of two;
 *   T > 0: two launches instead of three (rows of at most 256 sampling chunks of 256 16-byte
 *          vectors, i.e. 524288 bf16 / 262144 fp32 logits, and the num_seqs x chunks
 *          workgroups of the second launch resident at once with a quarter of the device to
 *          spare).
 * Every path gives identical results.  The single launches need their waiting workgroups
 * resident; a wait that gives up (after about a second, e.g. when other work holds the device)
 * writes -1: at T = 0 its sequence reports -1 in accept_len and next_token, at T > 0 in one or
 * both (an output that is not -1 is exact).
 * Errors: SD_ERR_INVALID_ARG, SD_ERR_WORKSPACE (smaller than the multi-launch path needs),
 * SD_ERR_HIP.  S == 0 returns SD_OK.
 */
int sd_accept(const sd_accept_shape *shape, const void *target_logits, const void *draft_logits,
              const int32_t *draft_tokens, const float *uniforms, const int32_t *block_lens,
              const int32_t *q_offsets, float temperature, int32_t *accept_len, int32_t *next_token,
              void *workspace, size_t workspace_bytes, void *stream);

/*
 * sd_accept without a workspace argument, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).  The
 * arguments, the kernels and the results are those of sd_accept; the scratch space is a fixed
 * array of SD_ACCEPT_NOALLOC_SCRATCH_BYTES in device memory that the library holds on each
 * device it runs on until the process ends.  Its address is looked up once per device, on the
 * first call made with that device current.  The call allocates nothing, and its scratch
 * needs no clearing (every byte a kernel reads was written earlier in the same call).
 *
 * Every call on one device shares that device's array: two calls that may run at the same
 * time on one device (different streams, or different host threads without ordering) race on
 * it and give undefined results.  Order them on one stream, or use sd_accept with a workspace
 * each.
 * Errors: as sd_accept; SD_ERR_WORKSPACE when the shape needs more scratch than the array holds
 * (sd_accept_workspace_size reports the need; about 2 * S * max_block * ceil(V / 32768) * 16
 * bytes at T > 0 with bf16 logits), SD_ERR_HIP if the array's address cannot be found.
 */
#define SD_ACCEPT_NOALLOC_SCRATCH_BYTES ((size_t)4 << 20)
int sd_accept_noalloc(const sd_accept_shape *shape, const void *target_logits, const void *draft_logits,
                      const int32_t *draft_tokens, const float *uniforms, const int32_t *block_lens,
                      const int32_t *q_offsets, float temperature, int32_t *accept_len, int32_t *next_token,
                      void *stream);

/*
 * Test hook for the acceptance paths of the calls enqueued after it, process-wide:
 *   mode 0 (default): the tagged-word launches where sd_accept's "Paths" allow them; 1: never.
 *   spin_limit > 0: polls before a wait of the single launch gives up; <= 0: the default.
 * Errors: SD_ERR_INVALID_ARG for another mode.
 */
int sd_accept_set_path(int32_t mode, int32_t spin_limit);

/* ==========================================================================
 * Checks of the per-sequence values the calls above read from device memory and take on
 * trust.  For tests and debugging, not for the hot path: one small launch files an error
 * word; nothing else is touched.  An element is read only where the values checked before
 * it keep the index inside its documented array.
 * ========================================================================== */
enum {
  SD_CHECK_CTX = 1,      /* ctx_s outside [0, max_ctx] */
  SD_CHECK_BLOCK = 2,    /* B_s outside [0, max_block] (attention) or [1, max_block] (acceptance) */
  SD_CHECK_OFFSETS = 4,  /* q_offsets[0] != 0, q_offsets[s+1] - q_offsets[s] != B_s, q_offsets[S] !=
                            total_q, or an offset outside [0, total_q] */
  SD_CHECK_TOKEN = 8,    /* a drafted token outside [0, V) */
  SD_CHECK_UNIFORM = 16  /* a uniform outside [0, 1), NaN included */
};

/*
 * status [3] int32 device out: status[0] = OR of the SD_CHECK_* bits found over all
 * sequences (0: the values meet sd_block_attn's documented ranges for this shape);
 * status[1] = the smallest offending sequence, or -1; status[2] = the number of offending
 * sequences.  ctx_lens, block_lens [S] and q_offsets [S + 1] as in sd_block_attn (may be
 * NULL when S == 0; status is still written).  Only num_seqs, total_q, max_ctx and max_block
 * of the shape are used.
 * Errors: SD_ERR_INVALID_ARG, SD_ERR_HIP.
 */
int sd_check_attn_inputs(const sd_attn_shape *shape, const int32_t *ctx_lens, const int32_t *block_lens,
                         const int32_t *q_offsets, int32_t *status, void *stream);

/*
 * The same for sd_accept: block_lens, q_offsets, draft_tokens [total_q - S] and, when
 * temperature > 0, uniforms [total_q] (unused and may be NULL at temperature 0).  Only
 * num_seqs, vocab, total_q and max_block of the shape are used.
 * Errors: SD_ERR_INVALID_ARG, SD_ERR_HIP.
 */
int sd_check_accept_inputs(const sd_accept_shape *shape, const int32_t *draft_tokens, const float *uniforms,
                           const int32_t *block_lens, const int32_t *q_offsets, float temperature,
                           int32_t *status, void *stream);

/* ==========================================================================
 * The step around verification.  One speculative step writes the block's keys and
 * values, verifies the block in every layer, accepts the longest consistent prefix
 * and commits it (Sec. 2.1; Fig. 1 caption).  The block size of a sequence is fixed
 * for the whole decoding (Sec. 2.4), so block_lens and q_offsets do not change from
 * step to step; only ctx_lens advances, on the device, with no host round trip.
 * ========================================================================== */

/*
 * k_cache[s, h, ctx_s + i, :] = k_new[q_offsets[s] + i, h, :] and the same for v, for every
 * block position i < B_s and kv head h.
 *
 *   k_new, v_new    [total_q, Hkv, D]   dtype (shape->dtype); the block's new keys and values
 *   k_cache,v_cache [S, Hkv, Lmax, D]   dtype, written in place
 *   ctx_lens        [S] int32           committed length before this step
 *   q_offsets       [S + 1] int32       exclusive prefix sum of the block lengths
 * Only num_seqs, num_q_heads, num_kv_heads, head_dim, max_kv_len, total_q and dtype of the
 * shape are used.  A row that would land at or past Lmax (ctx_s + i >= Lmax) is skipped, not
 * written.  Buffers 16-byte aligned.  Errors: SD_ERR_INVALID_ARG, SD_ERR_UNSUPPORTED, SD_ERR_HIP.
 */
int sd_kv_append(const sd_attn_shape *shape, const void *k_new, const void *v_new, void *k_cache, void *v_cache,
                 const int32_t *ctx_lens, const int32_t *q_offsets, void *stream);

/*
 * sd_kv_append into page pools (layout as in sd_block_attn_paged): block row i of sequence s
 * goes to logical key ctx_s + i.  A row past max_pages * page_size, or whose page id lies
 * outside [0, num_pages), is skipped, not written.  The shape's max_kv_len is not used.
 */
int sd_kv_append_paged(const sd_attn_shape *shape, int32_t page_size, int32_t num_pages, int32_t max_pages,
                       const int32_t *block_table, const void *k_new, const void *v_new, void *k_pages, void *v_pages,
                       const int32_t *ctx_lens, const int32_t *q_offsets, void *stream);

/*
 * ctx_lens[s] += accept_len[s] + 1: the block's anchor and its accepted drafts are now part of
 * the cached context.  Rows of rejected drafts remain past the new length and are overwritten by
 * the next sd_kv_append, so no rollback work is needed.  Both arrays are device int32 [S].
 * Errors: SD_ERR_INVALID_ARG, SD_ERR_HIP.
 */
int sd_commit(int32_t num_seqs, const int32_t *accept_len, int32_t *ctx_lens, void *stream);

/* Device buffers of one layer for sd_verify_step (a host array of these is passed). */
typedef struct sd_layer_buffers {
  const void *q;     /* [total_q, Hq, D]      queries of the block rows */
  const void *k_new; /* [total_q, Hkv, D]     the block's new keys */
  const void *v_new; /* [total_q, Hkv, D]     the block's new values */
  void *k_cache;     /* [S, Hkv, Lmax, D]     this layer's caches */
  void *v_cache;
  void *out;         /* [total_q, Hq, D]      attention output */
} sd_layer_buffers;

/* Workspace bytes sd_verify_step needs: the larger of the two operations' (host-only). */
int sd_verify_step_workspace_size(const sd_attn_shape *attn_shape, const sd_accept_shape *accept_shape,
                                  float temperature, size_t *bytes);

/*
 * One verify step, enqueued on `stream` with no host synchronisation: for every layer l,
 * sd_kv_append then sd_block_attn (layers[l]; for bf16 both in one sd_block_attn_append
 * launch); then sd_accept on the given logits; then
 * sd_commit (ctx_lens advances by accept_len + 1).  The logits are the caller's (the model's
 * head after the last layer); every other argument has the meaning given above.  The two
 * shapes must agree on num_seqs, total_q and max_block; attn_shape->max_ctx bounds ctx_lens
 * before the step.  All pointers are checked before any work is enqueued.
 * Errors: those of the four calls, SD_ERR_WORKSPACE.
 */
int sd_verify_step(const sd_attn_shape *attn_shape, int32_t num_layers, const sd_layer_buffers *layers,
                   int32_t *ctx_lens, const int32_t *block_lens, const int32_t *q_offsets, int32_t mask_mode,
                   const sd_accept_shape *accept_shape, const void *target_logits, const void *draft_logits,
                   const int32_t *draft_tokens, const float *uniforms, float temperature, int32_t *accept_len,
                   int32_t *next_token, void *workspace, size_t workspace_bytes, void *stream);

/* ==========================================================================
 * Block-size policy, run once per prompt after prefill (Sec. 2.3-2.4, Eq. 9).  The
 * predictive distribution of the prompt's last token, p = softmax(z), feeds an MLP
 * with two hidden layers (width 2048 by default, Sec. 3.1) scoring the 2k+1
 * candidate block sizes {B-k, ..., B+k}; the chosen size is the argmax:
 *   h1 = relu(W1 p + b1), h2 = relu(W2 h1 + b2), o = W3 h2 + b3,
 *   block_size = B - k + argmax_c o_c   (lowest c on ties).
 * ========================================================================== */
typedef struct sd_policy_shape {
  int32_t num_prompts;  /* P >= 0 */
  int32_t vocab;        /* V, a multiple of 8 */
  int32_t hidden;       /* H, a multiple of 8 (2048 in the paper) */
  int32_t radius;       /* k: 2k+1 <= 64 candidates */
  int32_t base_block;   /* B, the training block size; B - k >= 1 */
  int32_t logits_dtype; /* SD_BF16 or SD_F32 */
} sd_policy_shape;

/* Workspace bytes sd_block_size_policy needs (host-only). */
int sd_policy_workspace_size(const sd_policy_shape *shape, size_t *bytes);

/*
 *   last_logits  [P, V]     logits_dtype: the target's logits at each prompt's last position
 *   w1 [H, V], w2 [H, H], w3 [2k+1, H]   bf16, row-major (output dimension first)
 *   b1 [H], b2 [H], b3 [2k+1]            fp32
 *   scores       [P, 2k+1]  fp32 out: o
 *   block_size   [P] int32 out
 * p and the layer activations are fp32; products accumulate in fp32.  Logits and w1, w2, w3
 * 16-byte aligned; workspace 256-byte aligned, >= sd_policy_workspace_size().
 * Errors: SD_ERR_INVALID_ARG, SD_ERR_UNSUPPORTED (vocab or hidden not a multiple of 8),
 * SD_ERR_WORKSPACE, SD_ERR_HIP.  P == 0 returns SD_OK without touching the device.
 */
int sd_block_size_policy(const sd_policy_shape *shape, const void *last_logits, const void *w1, const float *b1,
                         const void *w2, const float *b2, const void *w3, const float *b3, float *scores,
                         int32_t *block_size, void *workspace, size_t workspace_bytes, void *stream);


/* ==========================================================================
 * Prefix-survival model of the accepted length (App. A).  For a sample x, block size
 * b and drafter training block size B:
 *   q_j(x, b)   = gamma_j(x) r(b; B),  r(b; B) = exp(-alpha (b - B)^2)       (App. A.2)
 *   tau(b; x)   = E[L_b(x)] = sum_{i=1..b} prod_{j=1..i} q_j(x, b)          (App. A.1)
 *   B*(x)       = argmax of tau over the candidates (smallest b on ties)     (App. A.2)
 *   R(x)        = tau(B*(x); x) - tau(B_hat(x); x)                           (App. A.3)
 *   L_tau(x)    = max over candidate pairs of |tau(b1) - tau(b2)| / |b1 - b2|: the smallest
 *                 constant of the discrete Lipschitz condition, so R(x) <= L_tau |B* - B_hat|.
 * gamma_j(x) is the intrinsic predictability of drafted position j (App. A.2).  Arithmetic
 * is fp64.  No workspace; nothing is allocated.
 * ========================================================================== */
typedef struct sd_survival_shape {
  int32_t num_samples; /* N >= 0 */
  int32_t max_pos;     /* P: positions per sample in gamma, 1..128 */
  int32_t num_cands;   /* C: 1..64 */
  int32_t train_block; /* B */
  double alpha;        /* retention sharpness, finite and >= 0 */
  int32_t cands[64];   /* host: the C candidate block sizes, strictly ascending, each in [1, P] */
} sd_survival_shape;

/*
 *   gamma      [N, P] fp32 device, 16-byte aligned: gamma_j(x) of sample n at column j - 1
 *   b_hat      [N] int32 device or NULL: a predicted block size per sample
 *   tau        [N, C] fp64 device out: tau(cands[c]; x_n)
 *   b_star     [N] int32 device out: B*(x_n)
 *   regret     [N] fp64 device out (given exactly when b_hat is): R(x_n); NaN where b_hat[n]
 *              is not a candidate
 *   lipschitz  [N] fp64 device out or NULL: L_tau(x_n)
 * Errors: SD_ERR_INVALID_ARG, SD_ERR_HIP.  N == 0 returns SD_OK without touching the device.
 */
int sd_survival_tau(const sd_survival_shape *shape, const float *gamma, const int32_t *b_hat, double *tau,
                    int32_t *b_star, double *regret, double *lipschitz, void *stream);

/*
 * Monte Carlo of L_b(x): `trials` independent verification passes per (sample, candidate).
 * Drafted position i (1-based) of trial t, candidate index c, sample n is accepted iff
 * u < q_i(x, b), with u the top 53 bits over 2^53 of word (i-1) mod 4 of Philox4x64-10
 * (Salmon et al., SC'11) under key (seed, 0) at counter ((i-1) div 4, t, c, n); L is the
 * number of leading acceptances, so L <= b.  The draws depend on those indices only, not on
 * the launch.
 *   mean_len  [N, C] fp64 device out: (sum of L over the trials) / trials
 *   len_hist  [N, C, P + 1] int32 device out or NULL: trials with L = 0..P
 * trials in [1, 2^30].  Errors: SD_ERR_INVALID_ARG, SD_ERR_HIP.
 */
int sd_survival_sample(const sd_survival_shape *shape, const float *gamma, uint64_t seed, int32_t trials,
                       double *mean_len, int32_t *len_hist, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* SD_BLOCK_H */
