/*
 * dvs.h - C ABI of the self-speculative draft-verify step for MI355X (gfx950).
 *
 * One step of self-speculative decoding (method section "Self-Speculative
 * Decoding" and the appendix "Self-Speculative Decoding and KV-Cache
 * Update") carried out in a single forward of R = n_causal + n_mask window
 * rows per sequence:
 *
 *   causal rows  r = 0..n_causal-1 : inputs [x0, d_1..d_{n_causal-1}],
 *                                     token-level causal attention (verify);
 *   mask rows    r = n_causal..R-1 : the mask token [M], attending to the
 *                                     whole cache, every causal row and,
 *                                     bidirectionally, the whole mask block
 *                                     (block diffusion draft; Preliminaries
 *                                     "Block Diffusion").
 *
 * The hot path is attn_hybrid_block -> argmax_accept -> kv_commit;
 * draft_verify_step runs a whole decoder forward plus those stages.
 *
 * Conventions for every entry point
 *   - All array arguments are DEVICE pointers owned by the caller.  The
 *     library never allocates or frees device memory in these calls; scratch
 *     space is passed in as `workspace` and sized by the *_workspace_bytes
 *     queries.  Arrays are dense, row-major, with the shapes given below.
 *   - `stream` is a hipStream_t (NULL = the null stream).  Every call only
 *     enqueues work on it and returns without synchronising.
 *   - Return value: DVS_OK, or a negative DVS_E* code when the host-side
 *     argument check fails (then nothing is launched) or a launch fails.
 *     dvs_last_error() gives a message for the calling thread.
 *   - Conditions that only the device can see (bad page ids, pool
 *     exhaustion, non-finite logits, ...) OR a DVS_ERR_* bit into the
 *     caller's int32 `err_word` (device memory, never cleared by the
 *     library); the affected sequences are left unmodified.
 *   - Page size is fixed at 16 tokens.  K pools are laid out
 *     [num_pool_pages, Hkv, 16, D] and V pools head-dim-major
 *     [num_pool_pages, Hkv, D, 16]; logical position p of sequence s lives in
 *     page page_table[s * max_pages + p / 16], slot p % 16.
 *   - dtype: DVS_F32 (float) or DVS_BF16 (bfloat16 storage, fp32 accumulate).
 */
#ifndef DVS_H
#define DVS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DVS_OK 0
#define DVS_EINVAL (-1)        /* bad pointer, shape or parameter          */
#define DVS_EUNSUPPORTED (-2)  /* valid but not implemented (D, dtype, ...) */
#define DVS_EHIP (-3)          /* a HIP launch or query failed             */
#define DVS_EWORKSPACE (-4)    /* workspace missing or too small           */

#define DVS_F32 0
#define DVS_BF16 1

#define DVS_ERR_POOL_EXHAUSTED 1  /* commit needed more free pages than exist */
#define DVS_ERR_MAX_PAGES 2       /* a sequence would exceed max_pages        */
#define DVS_ERR_NONFINITE 4       /* a logit was NaN or infinite              */
#define DVS_ERR_BAD_PAGE 8        /* a page id outside [0, num_pool_pages)    */
#define DVS_ERR_OPEN_BLOCK 16     /* a block commit met a masked position     */

#define DVS_PAGE_SIZE 16

int dvs_version(void);
const char* dvs_last_error(void);

/* ------------------------------------------------------------------------
 * attn_hybrid_block
 *
 * Appends the window's K/V to the cache, then computes block-causal (hybrid)
 * masked softmax attention for every window row (Preliminaries "Block
 * Diffusion": causal across blocks, bidirectional within the block; Method
 * "Joint AR-Diffusion Training": a corrupted block sees the preceding clean
 * blocks and itself; appendix items Draft forward / Verify forward).
 *
 * For sequence s with committed length L = kv_len[s], window row r sits at
 * position L + r and sees key position k iff
 *     k <= L + r            for r <  n_causal   (token-level causal),
 *     k <= L + R - 1        for r >= n_causal   (cache + whole window).
 * out[s,r,h,:] = sum_k softmax_k(softmax_scale * <q[s,r,h], K_k>) V_k over the
 * visible keys, with query head h reading KV head h / (Hq / Hkv).
 *
 *   q       [S, R, Hq, D]     window queries (after any position encoding)
 *   k_new   [S, R, Hkv, D]    window keys, written to positions [L, L+R)
 *   v_new   [S, R, Hkv, D]    window values, written likewise
 *   k_pool  [num_pool_pages, Hkv, 16, D]  paged K cache (updated)
 *   v_pool  [num_pool_pages, Hkv, D, 16]  paged V cache, head-dim-major (updated)
 *   page_table [S, max_pages] int32, kv_len [S] int32 (read only)
 *   out     [S, R, Hq, D]     attention output, same dtype as q
 *   chunk_keys   key-range split per workgroup (multiple of 64), or 0 for
 *                the balanced split.  Chunks start at absolute positions that
 *                are multiples of it, so a row's arithmetic does not depend on
 *                the other rows (a causal row equals an AR call bit for bit).
 *                0: the items' tiles are shared out evenly over the chip,
 *                whatever the length mix; a row's rounding then depends on
 *                the call's other rows, which drops that bit-equality.
 *   err_word     int32 device word (may be NULL): DVS_ERR_MAX_PAGES if
 *                L + R > max_pages * 16, DVS_ERR_BAD_PAGE for a page id
 *                outside the pool; such sequences are skipped.
 *   workspace    >= dvs_attn_workspace_bytes(...) bytes of device memory,
 *                zero-filled before its first call with a given shape (S, R,
 *                heads, D, max_pages, chunk_keys); its leading bytes are
 *                split-merge counters that every call leaves zero again, so
 *                later calls of the same shape need no clearing.
 *                Calls that share a workspace must not overlap in time.
 * Requirements: Hq % Hkv == 0, D in {64, 96, 128}, R >= 1, S >= 1, all
 * pointers non-NULL (except err_word), softmax_scale > 0.
 * ---------------------------------------------------------------------- */
size_t dvs_attn_workspace_bytes(int32_t S, int32_t n_causal, int32_t n_mask, int32_t Hq,
                                int32_t Hkv, int32_t D, int32_t max_pages, int32_t chunk_keys,
                                int32_t dtype);

int attn_hybrid_block(const void* q, const void* k_new, const void* v_new, void* k_pool,
                      void* v_pool, const int32_t* page_table, const int32_t* kv_len,
                      int32_t S, int32_t n_causal, int32_t n_mask, int32_t Hq, int32_t Hkv,
                      int32_t D, int32_t max_pages, int32_t num_pool_pages,
                      float softmax_scale, int32_t dtype, int32_t chunk_keys, void* out,
                      int32_t* err_word, void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * attn_hybrid_block_grouped
 *
 * attn_hybrid_block with the mask rows cut into groups of mask_group rows
 * (0: one group, which is attn_hybrid_block).  With G = n_mask / mask_group
 * groups (G <= n_causal), row i of mask group g sees the cache, the causal
 * rows 0 .. n_causal - G + g and, bidirectionally, the rows of its own group
 * (window slots [L + n_causal + g*mask_group, L + n_causal + (g+1)*mask_group));
 * causal rows are unchanged.  With G = n_causal = B and B rows per group,
 * group k is the draft block of the continuation that keeps the causal rows
 * 0..k: one draft per possible acceptance length, the structured-mask
 * AR-diffusion hybrid the paper cites in its related work (multidraft_step).
 * The window's K/V is appended at [L, L + R) in row order as before; query
 * positions (rotary) are the caller's.  Workspace as attn_hybrid_block.
 * ---------------------------------------------------------------------- */
int attn_hybrid_block_grouped(const void* q, const void* k_new, const void* v_new, void* k_pool,
                              void* v_pool, const int32_t* page_table, const int32_t* kv_len,
                              int32_t S, int32_t n_causal, int32_t n_mask, int32_t mask_group,
                              int32_t Hq, int32_t Hkv, int32_t D, int32_t max_pages,
                              int32_t num_pool_pages, float softmax_scale, int32_t dtype,
                              int32_t chunk_keys, void* out, int32_t* err_word, void* workspace,
                              size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * attn_hybrid_block_noalloc
 *
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  The same
 * computation, arguments and error behaviour as attn_hybrid_block, without
 * the workspace: the split partials and counters live in a device array of
 * DVS_ATTN_SCRATCH_BYTES inside the library, one per GPU, held from the
 * library's first use on that GPU until the process ends.  The call
 * allocates nothing (no hipMalloc, hipFree or allocating library routine);
 * it clears the counters it uses with a kernel on `stream` first.
 *   - A shape whose attn_hybrid_block workspace (dvs_attn_workspace_bytes)
 *     exceeds DVS_ATTN_SCRATCH_BYTES is rejected with DVS_EWORKSPACE before
 *     anything is launched; the fp32 path needs no scratch.
 *   - Every call on one GPU shares that GPU's array: calls that overlap in
 *     time on one GPU (other streams, other host threads) race and give
 *     wrong results; serialise them.
 *   - DVS_EHIP if the array's device address cannot be obtained.
 * ---------------------------------------------------------------------- */
#define DVS_ATTN_SCRATCH_BYTES (64u << 20)

int attn_hybrid_block_noalloc(const void* q, const void* k_new, const void* v_new, void* k_pool,
                              void* v_pool, const int32_t* page_table, const int32_t* kv_len,
                              int32_t S, int32_t n_causal, int32_t n_mask, int32_t Hq,
                              int32_t Hkv, int32_t D, int32_t max_pages, int32_t num_pool_pages,
                              float softmax_scale, int32_t dtype, int32_t chunk_keys, void* out,
                              int32_t* err_word, void* stream);

/* ------------------------------------------------------------------------
 * argmax_accept
 *
 * Top-1 over the vocabulary for every window row, then greedy acceptance
 * (method "Self-Speculative Decoding"; appendix item Accept):
 *   argmax_out[s, r] = index of the largest logits[s, r, :]; among equal
 *                      maxima the lowest index; -0.0 equals +0.0;
 *   a_j = argmax_out[s, j-1]  (row j-1 predicts the token after it);
 *   accept_len[s] = A = largest k <= n_causal-1 with draft[s, j-1] == a_j
 *                   for every j <= k.
 *
 *   logits   [S, R, V]  DVS_F32 or DVS_BF16
 *   draft    [S, draft_width] int32; draft_width >= n_causal - 1
 *   argmax_out [S, R] int32, accept_len [S] int32 (written); accept_len
 *             may be NULL: then only the top-1 is computed (for
 *             accept_commit, which accepts inside the commit kernel)
 *   err_word  DVS_ERR_NONFINITE if any logit is NaN/Inf.  May be NULL.  Such
 *             a row still gets a vocabulary index: NaN values never win, so
 *             the top-1 is taken over the other values; a row with no value
 *             above -inf gives the lowest index holding -inf, or 0 when every
 *             value is NaN.
 * Requirements: 1 <= n_causal <= R, V >= 1.
 * ---------------------------------------------------------------------- */
int argmax_accept(const void* logits, int32_t dtype, int32_t S, int32_t R, int32_t V,
                  int32_t n_causal, const int32_t* draft, int32_t draft_width,
                  int32_t* argmax_out, int32_t* accept_len, int32_t* err_word, void* stream);

/* ------------------------------------------------------------------------
 * top1_confidence
 *
 * Top-1 and its softmax probability for every row (appendix "Direct
 * Block-Diffusion Decoding": a prediction is revealed by its token
 * probability):
 *   argmax_out[r] = top-1 of logits[r, :] (the rule of argmax_accept);
 *   conf_out[r]   = exp(z_max) / sum_i exp(z_i) = 1 / sum_i exp(z_i - z_max),
 *                   fp32 arithmetic, one pass over the row.
 *   logits [rows, V] DVS_F32 or DVS_BF16; argmax_out [rows] int32 and
 *   conf_out [rows] fp32 (written); err_word: DVS_ERR_NONFINITE as in
 *   argmax_accept (may be NULL); a row with no value above -inf gets the
 *   index rule of argmax_accept and confidence 0.
 * ---------------------------------------------------------------------- */
int top1_confidence(const void* logits, int32_t dtype, int32_t rows, int32_t V,
                    int32_t* argmax_out, float* conf_out, int32_t* err_word, void* stream);

/* ------------------------------------------------------------------------
 * kv_commit
 *
 * Commit and KV rollback for one step (appendix items Accept, Cache update,
 * Next round).  For every sequence s with finished[s] == 0:
 *   run      = d_1..d_A, a_{A+1}   (A = accept_len[s], a_j = argmax[s, j-1]);
 *   kept     = run truncated after the first eos_id (inclusive; eos_id < 0 =
 *              none) and at max_new total output tokens; k = |kept| >= 1;
 *   out_tokens[s, out_count[s] ...] += kept;  out_count[s] += k;
 *   kv_len[s] += k  (KV of x0 and the accepted drafts is kept; every other
 *                    window slot, including all mask-row slots, is dropped);
 *   boundary[s] = last kept token;
 *   draft[s, j-1] = argmax[s, n_causal + j - 1], j = 1..draft_width, when
 *                   n_mask > 0 (requires n_mask >= draft_width);
 *   finished[s] = 1 when EOS was kept or max_new was reached.
 * Finished sequences are left unchanged.  Afterwards every sequence holds
 * exactly ceil((kv_len + R) / 16) pages: surplus pages are pushed onto the
 * free stack (sequences in order, highest logical page first), then missing
 * pages are popped from its top (sequences in order, logical pages
 * ascending); freed table entries become -1.  If the pops exceed the free
 * pages, or a table would exceed max_pages, NOTHING is changed and
 * DVS_ERR_POOL_EXHAUSTED / DVS_ERR_MAX_PAGES is ORed into err_word.
 *
 *   accept_len [S], argmax [S, R] (read)
 *   kv_len [S], page_table [S, max_pages], num_pages [S],
 *   free_stack [num_pool_pages], free_top [1], boundary [S],
 *   draft [S, draft_width], out_tokens [S, max_new], out_count [S],
 *   finished [S]  (all int32, read and written)
 * Requirements: 1 <= S <= 1024, 1 <= n_causal, 0 <= n_mask.
 * ---------------------------------------------------------------------- */
int kv_commit(int32_t S, int32_t n_causal, int32_t n_mask, const int32_t* accept_len,
              const int32_t* argmax, int32_t* kv_len, int32_t* page_table, int32_t* num_pages,
              int32_t max_pages, int32_t* free_stack, int32_t* free_top, int32_t num_pool_pages,
              int32_t* boundary, int32_t* draft, int32_t draft_width, int32_t* out_tokens,
              int32_t* out_count, int32_t max_new, int32_t eos_id, int32_t* finished,
              int32_t* err_word, void* stream);

/* ------------------------------------------------------------------------
 * accept_commit
 *
 * Acceptance, commit and KV rollback in one kernel (method "Self-Speculative
 * Decoding"; appendix items Accept, Cache update, Next round): for every
 * live sequence, A = largest k <= n_causal-1 with draft[s, j-1] ==
 * argmax[s, j-1] for every j <= k (the rule of argmax_accept), written to
 * accept_out[s] (0 for finished sequences; accept_out may be NULL); then
 * exactly kv_commit with that A.  Arguments, layouts, errors and
 * requirements as kv_commit, with argmax from argmax_accept (which may then
 * skip its own acceptance: accept_len = NULL).
 *   draft_group  0: the next draft is the mask rows' top-1, as kv_commit;
 *                > 0: the mask rows are n_causal groups of draft_group rows
 *                (attn_hybrid_block_grouped) and the next draft is group A's:
 *                draft[s, j-1] = argmax[s, n_causal + A*draft_group + j - 1].
 *                Needs n_mask == n_causal * draft_group >= draft_width.
 * ---------------------------------------------------------------------- */
int accept_commit(int32_t S, int32_t n_causal, int32_t n_mask, int32_t draft_group,
                  const int32_t* argmax,
                  int32_t* accept_out, int32_t* kv_len, int32_t* page_table, int32_t* num_pages,
                  int32_t max_pages, int32_t* free_stack, int32_t* free_top,
                  int32_t num_pool_pages, int32_t* boundary, int32_t* draft, int32_t draft_width,
                  int32_t* out_tokens, int32_t* out_count, int32_t max_new, int32_t eos_id,
                  int32_t* finished, int32_t* err_word, void* stream);

/* ------------------------------------------------------------------------
 * kv_commit_round
 *
 * The commit of the paper's two-forward round (appendix "Self-Speculative
 * Decoding and KV-Cache Update", items Accept, Cache update, Next round),
 * after a verify forward over [a0, d_1..d_B] (n_causal = B + 1, no mask
 * rows).  Same as kv_commit with R = B + 1 except:
 *   run      = a0, d_1..d_A, a_{A+1}   (a0 = lead[s]; A = accept_len[s] <= B,
 *              a_j = argmax[s, j-1]; 2..B+2 tokens before truncation);
 *   kv_len[s] += k - 1  (kv_len already counts x0, kept from the draft
 *                        forward; a0 and the kept drafts add their slots);
 *   pages cover the next round's windows: ceil((kv_len + B + 2) / 16);
 *   draft is not changed (the next round drafts afresh).
 *   lead [S] int32 (read); argmax [S, B + 1]; other arrays as in kv_commit.
 * Requirements: 1 <= S <= 1024, B >= 1, draft_width >= B.
 * ---------------------------------------------------------------------- */
int kv_commit_round(int32_t S, int32_t B, const int32_t* lead, const int32_t* accept_len,
                    const int32_t* argmax, int32_t* kv_len, int32_t* page_table, int32_t* num_pages,
                    int32_t max_pages, int32_t* free_stack, int32_t* free_top,
                    int32_t num_pool_pages, int32_t* boundary, int32_t* draft,
                    int32_t draft_width, int32_t* out_tokens, int32_t* out_count,
                    int32_t max_new, int32_t eos_id, int32_t* finished, int32_t* err_word,
                    void* stream);

/* ------------------------------------------------------------------------
 * draft_verify_step
 *
 * One fused self-speculative step of a decoder (method "Self-Speculative
 * Decoding"; appendix "Self-Speculative Decoding and KV-Cache Update"): the
 * window rows are embedded -- causal rows [x0, d_1..d_{n_causal-1}] from
 * state->boundary / state->draft, mask rows as the mask-token embedding, row
 * `vocab` of the table (Method "AR-to-Diffusion Conversion") -- and run
 * through every layer:
 *     h = RMSNorm(x) * g_attn;  q, k, v = h Wq^T, h Wk^T, h Wv^T;
 *     rotate-half rotary embedding at position kv_len + r (theta rope_theta);
 *     o = attn_hybrid_block(q, k, v, layer pools);  x += o Wo^T;
 *     if ffn > 0: h = RMSNorm(x) * g_mlp;  x += (silu(h Wg^T) * (h Wu^T)) Wd^T
 * then logits = (RMSNorm(x) * g_final) Wlm^T, argmax_accept and kv_commit on
 * the state.  With (n_causal, n_mask) = (B, B) this is the fused step;
 * (1, 0) is one greedy AR step.
 *
 * Weights are row-major [out_features, in_features]; all live in device
 * memory, in the model dtype (DVS_F32 or DVS_BF16; fp32 accumulation, fp32
 * residual stream, fp32 logits).  A row's arithmetic does not depend on how
 * many rows the call carries, so AR and fused calls agree bit for bit on the
 * causal rows (for the attention this needs chunk_keys > 0).
 *
 * logits_out [S*R, vocab] float, argmax_out [S*R], accept_out [S] int32 are
 * optional (NULL = kept in the workspace).  workspace: at least
 * dvs_step_workspace_bytes() bytes; no initialisation needed (the call clears
 * what must start at zero), and it may be shared with dvs_prefill.
 * ---------------------------------------------------------------------- */
typedef struct dvs_layer {
  const void* wq;      /* [n_heads*head_dim, hidden]        */
  const void* wk;      /* [n_kv_heads*head_dim, hidden]     */
  const void* wv;      /* [n_kv_heads*head_dim, hidden]     */
  const void* wo;      /* [hidden, n_heads*head_dim]        */
  const void* g_attn;  /* [hidden] RMSNorm gain             */
  const void* g_mlp;   /* [hidden]       (ffn > 0 only)     */
  const void* w_gate;  /* [ffn, hidden]  (ffn > 0 only)     */
  const void* w_up;    /* [ffn, hidden]  (ffn > 0 only)     */
  const void* w_down;  /* [hidden, ffn]  (ffn > 0 only)     */
  void* k_pool;        /* [num_pool_pages, n_kv_heads, 16, head_dim] */
  void* v_pool;        /* [num_pool_pages, n_kv_heads, head_dim, 16] */
} dvs_layer;

typedef struct dvs_model {
  int32_t dtype;       /* DVS_F32 or DVS_BF16 */
  int32_t n_layers, vocab, hidden, n_heads, n_kv_heads, head_dim, ffn;
  float rope_theta, rms_eps;
  const void* embed;   /* [vocab + 1, hidden]; row vocab = mask token [M] */
  const void* g_final; /* [hidden] */
  const void* lm_head; /* [vocab, hidden] */
  const dvs_layer* layers; /* HOST array of n_layers descriptors */
} dvs_model;

typedef struct dvs_state {
  int32_t S, max_pages, num_pool_pages, draft_width, max_new, eos_id;
  int32_t* kv_len;     /* [S]                 */
  int32_t* page_table; /* [S, max_pages]      */
  int32_t* num_pages;  /* [S]                 */
  int32_t* free_stack; /* [num_pool_pages]    */
  int32_t* free_top;   /* [1]                 */
  int32_t* boundary;   /* [S] x0              */
  int32_t* draft;      /* [S, draft_width]    */
  int32_t* out_tokens; /* [S, max_new]        */
  int32_t* out_count;  /* [S]                 */
  int32_t* finished;   /* [S]                 */
  int32_t* err_word;   /* [1] (may be NULL)   */
} dvs_state;

size_t dvs_step_workspace_bytes(const dvs_model* m, int32_t S, int32_t n_causal, int32_t n_mask,
                                int32_t max_pages, int32_t chunk_keys);
/* ------------------------------------------------------------------------
 * kv_commit_block
 *
 * The commit of one block of direct block-diffusion decoding (appendix
 * "Direct Block-Diffusion Decoding"), after the cache-write forward over
 * [x0, b_1..b_{B-1}].  Same as kv_commit except:
 *   run      = b_1..b_B = block[s, 0..B-1] (all B positions revealed; a
 *              negative token in the kept part of a live sequence's run sets
 *              DVS_ERR_OPEN_BLOCK and nothing is changed);
 *   kv_len[s] += k;  pages cover the next denoising window:
 *              ceil((kv_len + B + 1) / 16);  draft is not changed.
 *   block [S, B] int32 (read); other arrays as in kv_commit.
 * Requirements: 1 <= S <= 1024, B >= 1.
 * ---------------------------------------------------------------------- */
int kv_commit_block(int32_t S, int32_t B, const int32_t* block, int32_t* kv_len,
                    int32_t* page_table, int32_t* num_pages, int32_t max_pages,
                    int32_t* free_stack, int32_t* free_top, int32_t num_pool_pages,
                    int32_t* boundary, int32_t* out_tokens, int32_t* out_count, int32_t max_new,
                    int32_t eos_id, int32_t* finished, int32_t* err_word, void* stream);


int draft_verify_step(const dvs_model* m, const dvs_state* st, int32_t n_causal, int32_t n_mask,
                      int32_t chunk_keys, float* logits_out, int32_t* argmax_out,
                      int32_t* accept_out, void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * multidraft_step
 *
 * draft_verify_step with one draft block per possible acceptance length:
 * the window is the B causal rows [x0, d_1..d_{B-1}] followed by B groups
 * of B mask rows (R = B + B*B).  Group k assumes A = k: its rows sit at
 * positions L + k + 1 + i (i = 0..B-1; the first stands in for the
 * not-yet-known a_{k+1}, as the paper's draft forward puts [M] where a0
 * will be), attend to the cache, the causal rows 0..k and their own group
 * (attn_hybrid_block_grouped), and predict the tokens after d_1..d_k,
 * a_{k+1}.  Acceptance and commit are draft_verify_step's, except that the
 * next draft is group A's top-1 (accept_commit with draft_group = B), so it
 * is conditioned on the accepted drafts only -- never on a rejected one.
 * This is the structured-mask AR-diffusion hybrid of the paper's related
 * work, applied to the fused step; B = 1 is the fused step.  Group k's
 * outputs equal the mask rows of a fused call that verifies only x0,
 * d_1..d_k (n_causal = k + 1).
 * Pages must cover [L, L + B + B*B) (accept_commit leaves them so for the
 * next call); draft_width B - 1 or B.  logits_out [S*(B + B*B), vocab],
 * argmax_out [S*(B + B*B)], accept_out [S] optional as draft_verify_step.
 * workspace: dvs_step_workspace_bytes(m, S, B, B*B, max_pages, chunk_keys).
 * With chunk_keys > 0 every committed token equals greedy AR's bit for bit.
 * ---------------------------------------------------------------------- */
int multidraft_step(const dvs_model* m, const dvs_state* st, int32_t B, int32_t chunk_keys,
                    float* logits_out, int32_t* argmax_out, int32_t* accept_out,
                    void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * literal_round
 *
 * One round of the paper's two-forward self-speculative decoding (appendix
 * "Self-Speculative Decoding and KV-Cache Update"), with the layers of
 * draft_verify_step:
 *   1. draft forward over [x0, [M] x B] at positions L .. L+B (1 causal row,
 *      B mask rows): a0 = top-1 of the boundary row, d_j = top-1 of mask row
 *      j, written to state->draft[s, 0..B-1]; x0's causal KV is kept
 *      (kv_len + 1);
 *   2. verify forward over [a0, d_1..d_B] at positions L+1 .. L+B+1 (B + 1
 *      causal rows; its K/V overwrites the draft's mask-row slots):
 *      a_j = top-1 of row j-1, j = 1..B+1;
 *   3. A = longest prefix with d_j == a_j; kv_commit_round commits a0,
 *      d_1..d_A, a_{A+1} (2..B+2 tokens) and keeps pages for [L', L'+B+2).
 * Pages must cover [L, L + B + 2) on entry (kv_commit_round leaves them so;
 * after dvs_prefill the caller's page reservation must).  logits_out [S*(B+1), vocab]
 * receives the verify forward's logits, argmax_out [S*(B+1)] its top-1 and
 * accept_out [S] the accepted lengths (each optional).  workspace: at least
 * dvs_step_workspace_bytes(m, S, B + 1, 0, max_pages, chunk_keys) bytes.
 * With chunk_keys > 0 every committed token equals greedy AR's bit for bit.
 * ---------------------------------------------------------------------- */
int literal_round(const dvs_model* m, const dvs_state* st, int32_t B, int32_t chunk_keys,
                  float* logits_out, int32_t* argmax_out, int32_t* accept_out, void* workspace,
                  size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * diffusion_denoise / diffusion_block / dvs_diffusion_workspace_bytes
 *
 * Direct block-diffusion decoding (appendix "Direct Block-Diffusion
 * Decoding"), with the layers of draft_verify_step.  block [S, B] int32
 * holds the revealed token of block position p = 1..B in column p-1, or -1
 * while masked.
 *
 * diffusion_denoise: one forward over [x0, b_1..b_B] at positions L .. L+B
 *   (boundary row causal, block rows bidirectional, masked positions as
 *   [M]); top-1 and confidence (top1_confidence) of every row; then for
 *   every live sequence with masked positions: each masked position p whose
 *   row p-1 has confidence > tau_c takes that row's top-1; if none does,
 *   the masked position of largest confidence (lowest p among ties) does.
 *   Revealed positions never change; kv_len is unchanged.  *n_open (device
 *   int32, written) = number of live sequences whose block is still open.
 *   logits_out [S*(B+1), vocab] fp32, argmax_out [S*(B+1)] int32,
 *   conf_out [S*(B+1)] fp32 receive the forward's rows (each optional).
 *   workspace: dvs_step_workspace_bytes(m, S, 1, B, ...) bytes suffice.
 *
 * diffusion_block: one whole block: fills block with -1, runs
 *   diffusion_denoise until no live block is open (at most B forwards, each
 *   followed by a 4-byte device-to-host read and a stream synchronisation),
 *   then the cache-write forward over [x0, b_1..b_{B-1}] (B causal rows, no
 *   LM head) and kv_commit_block.  *steps_out (host, optional) = denoising
 *   forwards; the block cost *steps_out + 1 forwards.  Pages must cover
 *   [L, L + B + 1) on entry (kv_commit_block leaves them so).  workspace:
 *   dvs_diffusion_workspace_bytes(m, S, B, max_pages, chunk_keys) bytes.
 * ---------------------------------------------------------------------- */
size_t dvs_diffusion_workspace_bytes(const dvs_model* m, int32_t S, int32_t B, int32_t max_pages,
                                     int32_t chunk_keys);
int diffusion_denoise(const dvs_model* m, const dvs_state* st, int32_t B, float tau_c,
                      int32_t* block, int32_t* n_open, int32_t chunk_keys, float* logits_out,
                      int32_t* argmax_out, float* conf_out, void* workspace, size_t ws_bytes,
                      void* stream);
int diffusion_block(const dvs_model* m, const dvs_state* st, int32_t B, float tau_c,
                    int32_t* block, int32_t chunk_keys, int32_t* steps_out, void* workspace,
                    size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * literal_round_refined
 *
 * literal_round with a multi-step draft (experiments, "Draft Schedule": a
 * draft-side confidence threshold tau_d sets how many denoising forwards
 * build the draft).  The B + 1 predictions of the draft window [x0, b_1..b_B]
 * (a0 from the boundary row, d_j from row j) are revealed like a diffusion
 * block (the rule of diffusion_denoise, threshold tau_d); revealed a0,
 * d_1..d_{B-1} replace the [M] inputs of rows 1..B in the next draft forward
 * (d_B has no input slot).  When every live draft is complete (at most
 * B + 1 forwards, each followed by a 4-byte device-to-host read and a stream
 * synchronisation), the round continues as literal_round steps 2 and 3.
 * tau_d = 0 gives the one-shot draft of literal_round.  *draft_steps_out
 * (host, optional) = draft forwards; the round cost *draft_steps_out + 1
 * forwards.  Arguments, page and output conventions as literal_round;
 * workspace: the larger of dvs_step_workspace_bytes(m, S, 1, B, ...) and
 * dvs_step_workspace_bytes(m, S, B + 1, 0, ...).
 * ---------------------------------------------------------------------- */
int literal_round_refined(const dvs_model* m, const dvs_state* st, int32_t B, float tau_d,
                          int32_t chunk_keys, float* logits_out, int32_t* argmax_out,
                          int32_t* accept_out, int32_t* draft_steps_out, void* workspace,
                          size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * literal_round_sampled / dvs_sampled_round_workspace_bytes
 *
 * literal_round under sampling at temperature T, with the standard
 * acceptance-rejection rule of speculative decoding, which keeps the
 * committed tokens distributed as the verifier's own samples (Preliminaries,
 * "Speculative Decoding").  Each row's distribution is softmax(z / T) (fp32).
 *   1. draft forward over [x0, [M] x B]: a0 is sampled from the boundary
 *      row with u[s, 0] (the verifier's own distribution at L + 1) and d_j
 *      from mask row j (q_j) with u[s, j], j = 1..B; x0's KV is kept;
 *   2. verify forward over [a0, d_1..d_B]: p_j from row j-1;
 *   3. d_j is accepted while u[s, B + j] * q_j(d_j) < p_j(d_j); A = number
 *      accepted; the final token is sampled with u[s, 2B + 1] from
 *      max(0, p_{A+1} - q_{A+1}) (normalised) if A < B, else from p_{B+1};
 *      kv_commit_round commits a0, d_1..d_A and the final token.
 * Sampling from weights w with uniform u takes the smallest index whose
 * running sum (index order) exceeds u * sum(w).
 *   u [S, 2B + 2] fp32 uniforms in [0, 1) (device, read; the caller draws
 *   them); temperature > 0.  logits_out [S*(B+1), vocab] (verify logits) and
 *   accept_out [S] are optional.  Pages as literal_round.  workspace:
 *   dvs_sampled_round_workspace_bytes(m, S, B, max_pages, chunk_keys).
 * ---------------------------------------------------------------------- */
size_t dvs_sampled_round_workspace_bytes(const dvs_model* m, int32_t S, int32_t B,
                                         int32_t max_pages, int32_t chunk_keys);
int literal_round_sampled(const dvs_model* m, const dvs_state* st, int32_t B, float temperature,
                          const float* u, int32_t chunk_keys, float* logits_out,
                          int32_t* accept_out, void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * dvs_prefill
 *
 * Prefill of a fresh sequence (appendix item State: the first boundary token
 * is produced by prefill).  The window is the P prefix rows (causal) followed
 * by n_mask mask rows (bidirectional block), at positions 0 .. P+n_mask-1, so
 * the prefix KV is cached and the mask rows give the first draft:
 *   row r < P takes embed[prefix_tokens[s, r]] when that id is in
 *   [0, vocab) and x_prefix[s, r, :] otherwise (e.g. vision-encoder outputs;
 *   fp32, [S, P, hidden]); either array may be NULL when unused.
 * Afterwards kv_len = P, boundary = top-1 of row P-1 (also appended to the
 * output as the first committed token), draft[j] = top-1 of mask row j.
 * kv_len must be 0 on entry and every sequence must already hold pages for
 * positions [0, P + max(n_mask, R of the next step)).  logits_out (optional)
 * receives [S, n_mask + 1, vocab] fp32 for rows P-1 .. P+n_mask-1.
 * ---------------------------------------------------------------------- */
size_t dvs_prefill_workspace_bytes(const dvs_model* m, int32_t S, int32_t P, int32_t n_mask,
                                   int32_t max_pages, int32_t chunk_keys);

int dvs_prefill(const dvs_model* m, const dvs_state* st, int32_t P, int32_t n_mask,
                const int32_t* prefix_tokens, const float* x_prefix, int32_t chunk_keys,
                float* logits_out, void* workspace, size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DVS_H */
