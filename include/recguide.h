/*
 * recguide.h -- C ABI of the MI355X (gfx950) draft-verify hot path of
 * RecGuide (Reciprocal Guidance for diffusion-AR self-speculation).
 *
 * One fused forward step of a shared-backbone self-speculation model runs,
 * per request, the verify rows of the previous draft block and the rows of
 * the next draft block in the same batch.  This library provides the three
 * data-parallel pieces of that step:
 *
 *   rg_draft_verify_attention  attention of those rows over a paged KV cache
 *                              with the hybrid mask of Eq. 1 (Sec. 3.1)
 *   rg_verify_accept           verifier argmax / entropy per row and greedy
 *                              first-mismatch acceptance per request
 *                              (Sec. 3.1; e_t of Sec. 5.2)
 *   rg_draft_confidence        draft confidence P_1st, top-2 margin
 *                              P_1st - P_2nd and entropy per draft row
 *                              (Sec. 4.1)
 *   rg_verify_and_confidence   the two logit passes above in one call
 *   rg_verify_and_confidence_noalloc
 *                              the same without a workspace, for callers that
 *                              cannot allocate
 *
 * and, for the predictive draft-verify overlap (Sec. 5.1, served as in
 * Sec. 5.3):
 *
 *   rg_multibranch_attention   the step's attention when the rows after the
 *                              verify rows are several branches (correction
 *                              and continuation drafts) that share the
 *                              canonical prefix, read once for all of them
 *   rg_plan_branches           risky positions and the branches to prepare
 *   rg_match_branches          which prepared branch a verification confirms
 *
 * and, for verification-guided block sizing (Sec. 5.2) with block-size
 * bucketed serving (Sec. 5.3):
 *
 *   rg_plan_block_sizes        each request's next draft block size from its
 *                              verification history, and the requests grouped
 *                              by that size
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - bf16 tensors are passed as their raw 16-bit patterns (uint16_t).
 * - Pointers documented as "device" must point to memory the GPU can read
 *   or write (hipMalloc / torch CUDA tensors); "host" pointers are read by
 *   the CPU during the call only and may be reused as soon as it returns.
 * - The caller owns every buffer, including the workspace.  The library
 *   allocates no device memory and keeps no mutable global state other than
 *   the static scratch of rg_verify_and_confidence_noalloc (one array per
 *   GPU, and its address per device); calls on different streams are
 *   independent provided they use distinct workspaces and outputs.
 * - Every call validates its arguments on the host first.  On a validation
 *   error it returns the error code, enqueues nothing and leaves every output
 *   untouched.  Otherwise it enqueues its kernels on `stream` (a hipStream_t,
 *   NULL = the default stream) and returns without synchronising; outputs are
 *   valid once the stream reaches that point.  A failed launch returns
 *   RG_ERR_HIP.
 * - Workspaces: size them with the matching *_workspace query (same
 *   arguments).  An attention workspace (rg_draft_verify_attention,
 *   rg_multibranch_attention) must be all zero before its first use; each
 *   call leaves it ready for the next one (its synchronisation words return
 *   to zero), so zeroing it once when it is allocated is enough.  The other
 *   workspaces need no initialisation.  Contents are otherwise meaningless
 *   after a call.  Two calls in flight at once must not share a workspace.
 * - Inputs must be finite, and logits of magnitude below 2^127 (about
 *   1.7e38): the vocabulary passes scale logits by log2(e), which must not
 *   overflow.  A masked vocabulary entry can hold e.g. -1e30.
 */
#ifndef RECGUIDE_H
#define RECGUIDE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RG_ABI_VERSION 7

typedef int32_t rg_status;
#define RG_OK 0
#define RG_ERR_NULL 1        /* a required pointer is NULL                     */
#define RG_ERR_SHAPE 2       /* sizes or offsets are inconsistent             */
#define RG_ERR_UNSUPPORTED 3 /* valid but not supported (head_dim, page size) */
#define RG_ERR_WORKSPACE 4   /* workspace NULL or smaller than required       */
#define RG_ERR_HIP 5         /* a HIP launch or runtime call failed           */
#define RG_ERR_WAIT 6        /* a one-launch wait gave up (that call's outputs are invalid) */

/* Version of this ABI (RG_ABI_VERSION of the built library). */
int32_t rg_abi_version(void);

/* Static description of a status code. */
const char* rg_status_string(rg_status status);

/* Largest number of requests planned into one attention launch; larger
 * batches are split into several launches by the library itself. */
#define RG_ATTN_MAX_REQS_PER_LAUNCH 128

/*
 * Ragged batch layout of one fused draft-verify step (attention).
 *
 * Request r has ctx_len[r] = L tokens already in its pages and
 * n_r = q_indptr[r+1] - q_indptr[r] new query rows: first n_verify[r] = V
 * verify rows (the previous draft block), then B = n_r - V rows of the next
 * draft block.  The K/V of all n_r new rows must already be written to the
 * request's pages, so its keys are positions 0 .. T-1 with T = L + n_r.
 *
 * Mask (Eq. 1 with prefix = context + verify rows, draft set = next block):
 * verify row i (0 <= i < V) sees keys j <= L + i; draft rows see all T keys.
 *
 * Paged cache, page size 16 tokens.  Token j of request r lives in slot
 * j % 16 of page page_indices[page_indptr[r] + j / 16]; the request must own
 * at least ceil(T / 16) pages.  Cache layouts (contiguous):
 *   k_cache [num_pages][num_kv_heads][16][head_dim]   token-major pages
 *   v_cache [num_pages][num_kv_heads][head_dim][16]   dimension-major pages
 * Slots and pages no request reads may hold anything, NaN included.
 *
 * Grouped-query attention: query head h reads KV head h / (Hq / Hkv).
 */
typedef struct rg_attn_layout {
  int32_t num_requests;   /* R >= 1                                          */
  int32_t num_q_heads;    /* Hq >= 1                                         */
  int32_t num_kv_heads;   /* Hkv >= 1, Hq % Hkv == 0                         */
  int32_t head_dim;       /* D: 64 or 128                                    */
  int32_t page_size;      /* must be 16                                      */
  int32_t num_pages;      /* pages in each cache pool                        */
  float sm_scale;         /* softmax scale; <= 0 selects 1/sqrt(D)           */
  const int32_t* q_indptr;     /* host [R+1], q_indptr[0] = 0, nondecreasing  */
  const int32_t* n_verify;     /* host [R], 0 <= n_verify[r] <= n_r           */
  const int32_t* ctx_len;      /* host [R], >= 0                              */
  const int32_t* page_indptr;  /* host [R+1], page_indptr[0] = 0, nondecr.    */
  const int32_t* page_indices; /* DEVICE [page_indptr[R]], each < num_pages   */
} rg_attn_layout;

/* Workspace bytes rg_draft_verify_attention needs for this layout (0 if no
 * request is split across several KV chunks).  Zero it before its first use
 * (see the conventions above). */
rg_status rg_draft_verify_attention_workspace(const rg_attn_layout* layout, size_t* bytes);

/*
 * Hybrid-mask attention of one fused draft-verify step.
 *
 *   q     DEVICE [q_indptr[R]][Hq][D] bf16
 *   out   DEVICE [q_indptr[R]][Hq][D] bf16, softmax(scale*q.k + mask) . v,
 *         fp32 accumulation, rounded to nearest even
 *   lse   DEVICE [q_indptr[R]][Hq] fp32 natural-log log-sum-exp of the
 *         scaled, masked scores, or NULL
 *   ws    DEVICE workspace of at least the queried size (may be NULL when
 *         that size is 0), zero before its first use.
 *
 * Requests whose keys are split over several KV chunks need their chunks'
 * partial results merged: by default a second kernel does it after the main
 * one.  With the environment variable RG_ATTN_PERSIST=1 such a launch runs
 * instead as one work-queue launch (the library's variant of mapping mixed
 * ragged attention work onto the compute units, Sec. 5.3): at most one work
 * group per compute unit takes the work items (request, KV head, column
 * group, chunk; costliest request first) and then the merge items, every one
 * of them from an atomic queue, and a merge item starts as soon as the
 * chunks it merges are done (a bounded wait: see
 * rg_draft_verify_attention_check).  It gives the same results within
 * rounding and measured slower on MI355X.  The workspace opens with the queue and per-merge counters, at the
 * same place and size for every layout, so one workspace (zeroed once) may
 * serve calls with different layouts one after another.  A launch with more
 * than 16384 merge items always uses the two kernels.
 */
rg_status rg_draft_verify_attention(const rg_attn_layout* layout, const uint16_t* q,
                                    const uint16_t* k_cache, const uint16_t* v_cache,
                                    uint16_t* out, float* lse, void* ws, size_t ws_bytes,
                                    void* stream);

/*
 * One-launch mode (RG_ATTN_PERSIST=1) only: whether a merge item's bounded
 * wait gave up in a call on this attention workspace since the last check.
 * A correct call never gives up (every chunk a merge item waits for is held
 * by a running work group); if one did, that call's outputs are not valid.
 * The kernel moves the flag to a report word in the workspace's
 * synchronisation words, so it does not carry over into later calls; this
 * call synchronises `stream`, reads the report word and clears it.
 *   RG_OK        no wait gave up (or the workspace never ran a one-launch call)
 *   RG_ERR_WAIT  a wait gave up
 *   RG_ERR_NULL / RG_ERR_WORKSPACE  ws is NULL / too small to hold the words
 *   RG_ERR_HIP   the synchronisation or a copy failed
 */
rg_status rg_draft_verify_attention_check(void* ws, size_t ws_bytes, void* stream);

/* Planning summary of an attention call (host only, no GPU work): used by
 * tests and tools to inspect how the batch is split. */
typedef struct rg_attn_plan_info {
  int32_t num_launches;     /* launches of the main kernel                   */
  int32_t chunk_keys;       /* keys per KV chunk                             */
  int64_t work_items;       /* (request, kv head, column group, chunk) items */
  int64_t split_requests;   /* requests whose keys span more than one chunk  */
  int64_t partial_columns;  /* partial rows written to the workspace         */
  int64_t workspace_bytes;
  int32_t persistent_launches; /* launches run as one work-queue launch      */
  int32_t sync_words;       /* int32 synchronisation words at sync_offset    */
  int64_t sync_offset;      /* their byte offset in the workspace (-1 without
                               a workspace); word 3 is nonzero after a call
                               whose merge item gave up waiting (never
                               expected; see rg_draft_verify_attention_check) */
} rg_attn_plan_info;
rg_status rg_draft_verify_attention_plan(const rg_attn_layout* layout, rg_attn_plan_info* info);

/*
 * Greedy verification (Sec. 3.1; greedy decoding as in Sec. 6.1).
 *
 *   logits        DEVICE [total_rows] rows of `vocab` bf16 values, row k at
 *                 logits + k * row_stride (row_stride >= vocab, elements)
 *   row_indptr    DEVICE [R+1] int32: request r owns verify rows
 *                 row_indptr[r] .. row_indptr[r+1]-1 (may be empty);
 *                 row_indptr[0] = 0, row_indptr[R] = total_rows
 *   draft_tokens  DEVICE [total_rows] int32: the token row k judges; a
 *                 negative token marks a bonus row that never matches
 * Outputs (DEVICE, int32 / fp32):
 *   row_argmax     [total_rows]  lowest index of the row maximum
 *   accept_len     [R]  first k < V_r with row_argmax != token, else V_r
 *   next_token     [R]  row_argmax of row accept_len, or -1 if all matched
 *   row_entropy    [total_rows] or NULL: entropy (nats) of softmax(row)
 *   accept_entropy [R] or NULL: mean row entropy over rows
 *                  0 .. min(accept_len, V_r - 1) (the e_t of Sec. 5.2);
 *                  requests without rows get accept_len 0, next_token -1,
 *                  accept_entropy 0.
 */
rg_status rg_verify_accept_workspace(int32_t num_requests, int32_t total_rows, int32_t vocab,
                                     size_t* bytes);
rg_status rg_verify_accept(const uint16_t* logits, int64_t row_stride, int32_t vocab,
                           int32_t num_requests, int32_t total_rows, const int32_t* row_indptr,
                           const int32_t* draft_tokens, int32_t* row_argmax, int32_t* accept_len,
                           int32_t* next_token, float* row_entropy, float* accept_entropy,
                           void* ws, size_t ws_bytes, void* stream);

/*
 * Draft confidence per row (Sec. 4.1), softmax at temperature 1.
 *
 *   logits  DEVICE [total_rows] rows of `vocab` bf16 values (vocab >= 2),
 *           row k at logits + k * row_stride
 * Outputs (DEVICE):
 *   top1    [rows] int32  lowest index of the maximum
 *   top2    [rows] int32  lowest index of the maximum over the other entries
 *   p1      [rows] fp32   P_1st = softmax(row)[top1]   (confidence C_i)
 *   p2      [rows] fp32   P_2nd = softmax(row)[top2]
 *   margin  [rows] fp32 or NULL  P_1st - P_2nd          (margin M_i)
 *   entropy [rows] fp32 or NULL  entropy (nats) of softmax(row)
 */
rg_status rg_draft_confidence_workspace(int32_t total_rows, int32_t vocab, size_t* bytes);
rg_status rg_draft_confidence(const uint16_t* logits, int64_t row_stride, int32_t vocab,
                              int32_t total_rows, int32_t* top1, int32_t* top2, float* p1,
                              float* p2, float* margin, float* entropy, void* ws,
                              size_t ws_bytes, void* stream);

/*
 * Both logit passes of one round (Sec. 3.1: one forward pass of the fused
 * step yields the verify rows of the previous block and the rows of the next
 * draft block) in two launches instead of four.  The results are bit for bit
 * those of rg_verify_accept(verify_logits, verify_stride, vocab,
 * num_requests, verify_rows, row_indptr, draft_tokens, row_argmax,
 * accept_len, next_token, row_entropy, accept_entropy, ...) followed by
 * rg_draft_confidence(draft_logits, draft_stride, vocab, draft_rows, top1,
 * top2, p1, p2, margin, entropy, ...); arguments, layouts and NULL rules as
 * there (vocab >= 2).  One DEVICE workspace of at least the queried size,
 * 256-byte aligned (RG_ERR_WORKSPACE otherwise).
 */
rg_status rg_verify_and_confidence_workspace(int32_t num_requests, int32_t verify_rows,
                                             int32_t draft_rows, int32_t vocab, size_t* bytes);
rg_status rg_verify_and_confidence(const uint16_t* verify_logits, int64_t verify_stride,
                                   const uint16_t* draft_logits, int64_t draft_stride, int32_t vocab,
                                   int32_t num_requests, int32_t verify_rows,
                                   const int32_t* row_indptr, const int32_t* draft_tokens,
                                   int32_t* row_argmax, int32_t* accept_len, int32_t* next_token,
                                   float* row_entropy, float* accept_entropy, int32_t draft_rows,
                                   int32_t* top1, int32_t* top2, float* p1, float* p2, float* margin,
                                   float* entropy, void* ws, size_t ws_bytes, void* stream);

/*
 * rg_verify_and_confidence without a workspace argument, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation).  Arguments, outputs and results
 * are exactly rg_verify_and_confidence's; the chunk states that call keeps in
 * the caller's workspace go to a static device array of
 * RG_NOALLOC_SCRATCH_BYTES bytes instead, of which every GPU the library runs
 * on holds one copy until the process ends (its address is looked up once
 * per device, on that device's first call).  No device memory is allocated
 * and no allocating library routine is called.  A round whose workspace
 * (rg_verify_and_confidence_workspace) would exceed the array returns
 * RG_ERR_UNSUPPORTED before anything is enqueued: e.g. at vocabulary 128256
 * up to about 6500 verify plus 6500 draft rows fit.  Nothing in the array has
 * to start at zero.  All calls on one GPU share its array: two calls whose
 * kernels may overlap (other streams, other threads) race on it and must be
 * ordered by the caller.
 */
#define RG_NOALLOC_SCRATCH_BYTES (4u << 20)
rg_status rg_verify_and_confidence_noalloc(const uint16_t* verify_logits, int64_t verify_stride,
                                           const uint16_t* draft_logits, int64_t draft_stride, int32_t vocab,
                                           int32_t num_requests, int32_t verify_rows, const int32_t* row_indptr,
                                           const int32_t* draft_tokens, int32_t* row_argmax, int32_t* accept_len,
                                           int32_t* next_token, float* row_entropy, float* accept_entropy,
                                           int32_t draft_rows, int32_t* top1, int32_t* top2, float* p1, float* p2,
                                           float* margin, float* entropy, void* stream);

/* ------------------------------------------------------------------------
 * Predictive draft-verify overlap (Sec. 5.1, Sec. 5.3)
 * ------------------------------------------------------------------------ */

/* Largest number of requests planned into one multi-branch attention launch
 * (larger batches are split into several launches by the library). */
#define RG_BRANCH_MAX_REQS_PER_LAUNCH 64

/*
 * Branches of each request of a step (host arrays, read during the call).
 *
 * Request r lists branches branch_indptr[r] .. branch_indptr[r+1]-1.  Its
 * query rows (rg_attn_layout) are its n_verify[r] = V verify rows
 * followed by each listed branch's rows in order, and its keys are its
 * ctx_len[r] = L cached tokens, the V verify rows, then the branch rows in
 * the same order (their K/V written to the request's pages like any token).
 * A branch k keeps the canonical prefix of the context and its first
 * prefix[k] verify rows, then has rows[k] rows of its own, the first lead[k]
 * of which are committed tokens (e.g. a correction token) and the rest a
 * draft block.  Mask (Eq. 1 applied to the branch's own sequence): a lead
 * row sees the kept prefix and the branch's rows up to itself; a draft row
 * sees the kept prefix and all of the branch's rows.  Verify row i sees keys
 * j <= L + i as in rg_draft_verify_attention; no row sees another branch.
 * A request listing no branch treats its rows after the verify rows as one
 * continuation block (prefix V, lead 0): exactly rg_draft_verify_attention.
 *
 *   branch_indptr  host [R+1], branch_indptr[0] = 0, nondecreasing
 *   prefix         host [branch_indptr[R]], 0 .. V (at most 4095)
 *   lead           host [branch_indptr[R]], 0 .. rows (at most 15)
 *   rows           host [branch_indptr[R]], >= 1 (at most 65535); the listed
 *                  rows of a request sum to its rows after the verify rows
 * A request may list any number of branches as long as all but at most two
 * leading ones form one regular family: equal rows and lead, prefixes growing
 * by a constant step >= 0 (up to 65535 branches, step at most 4095) -- e.g.
 * correction and continuation branches (up to three of any shape), or one
 * draft block per hypothetical accepted length 0 .. V (the quadratic layout
 * of Sec. 6.2's comparison).
 * Violations give RG_ERR_SHAPE; a list of another form or a value past its
 * packing limit RG_ERR_UNSUPPORTED.
 */
typedef struct rg_branch_layout {
  const int32_t* branch_indptr;
  const int32_t* prefix;
  const int32_t* lead;
  const int32_t* rows;
} rg_branch_layout;

/* Workspace bytes rg_multibranch_attention needs (same arguments). */
rg_status rg_multibranch_attention_workspace(const rg_attn_layout* layout,
                                             const rg_branch_layout* branches, size_t* bytes);

/*
 * Attention of a step whose rows after the verify rows are overlap branches
 * (Sec. 5.1) that share the canonical prefix: every key of a request,
 * prefix included, is read from HBM once for all its rows (the shared-prefix
 * access of Sec. 5.3), and only valid query rows are processed.  Tensors,
 * output, lse and workspace as in rg_draft_verify_attention.
 */
rg_status rg_multibranch_attention(const rg_attn_layout* layout, const rg_branch_layout* branches,
                                   const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                                   uint16_t* out, float* lse, void* ws, size_t ws_bytes, void* stream);

/*
 * Branches to prepare for each request's draft block (Sec. 5.1).
 *
 *   margin, top2   DEVICE [total_rows] draft margin P_1st - P_2nd and
 *                  second-ranked token of each draft row (rg_draft_confidence
 *                  outputs of the block's rows)
 *   row_indptr     DEVICE [R+1]: request r's block is rows row_indptr[r] ..
 *                  row_indptr[r+1]-1, at positions 0, 1, ... (at most 65535
 *                  rows per request)
 *   delta          positions with margin < delta are risky
 * Outputs (DEVICE, int32): n_risky [R] risky positions in the block;
 * n_corr [R] = min(n_risky, 2) correction branches; corr_pos [R][2] their
 * positions (the earliest two risky ones, ascending; -1 past n_corr);
 * corr_tok [R][2] the replacement token top2 there (-1 past n_corr);
 * continuation [R] 1 when a continuation branch is prepared (n_risky <= 2).
 */
rg_status rg_plan_branches(const float* margin, const int32_t* top2, const int32_t* row_indptr,
                           int32_t num_requests, int32_t total_rows, float delta, int32_t* n_risky,
                           int32_t* n_corr, int32_t* corr_pos, int32_t* corr_tok, int32_t* continuation,
                           void* stream);

/*
 * Which prepared branch each request's verification confirms (Sec. 5.1).
 *
 *   accept_len, next_token  DEVICE [R] rg_verify_accept outputs of the block
 *   block_len               DEVICE [R] draft tokens of the block (full
 *                           acceptance = accept_len == block_len, with
 *                           next_token then the verifier's bonus token)
 *   n_corr, corr_pos, corr_tok, continuation
 *                           DEVICE rg_plan_branches outputs for the block
 *   cont_first              DEVICE [R] first token of the continuation branch
 * Output reused [R] (DEVICE int32): c when correction branch c matched
 * (accept_len == corr_pos[r][c] and next_token == corr_tok[r][c]); n_corr[r]
 * (the continuation's place after the corrections) when the continuation
 * matched (full acceptance, next_token == cont_first[r]); -1 otherwise.
 */
rg_status rg_match_branches(const int32_t* accept_len, const int32_t* next_token, const int32_t* block_len,
                            const int32_t* n_corr, const int32_t* corr_pos, const int32_t* corr_tok,
                            const int32_t* continuation, const int32_t* cont_first, int32_t num_requests,
                            int32_t* reused, void* stream);

/* ------------------------------------------------------------------------
 * Verification-guided block sizing and bucketing (Sec. 5.2, Sec. 5.3)
 * ------------------------------------------------------------------------ */

#define RG_BLOCK_MAX_CANDIDATES 8
#define RG_BLOCK_MAX_S_BINS 64
#define RG_BLOCK_MAX_REQUESTS 65536

/*
 * The block-size policy of Eq. 3 at one serving load C.
 *
 *   num_candidates  NB, 1 .. 8
 *   candidates      host [NB] candidate block sizes, ascending, distinct, >= 1
 *   num_s_bins      NS, 1 .. 64: the table's s axis is cut into NS bins
 *   s_edges         host [NS-1] nondecreasing bin edges (NULL when NS = 1);
 *                   bin k holds s_edges[k-1] <= s < s_edges[k]
 *   cost            host [NB] profiled execution cost T_C(B) of each candidate
 *   rho             the cost weight rho_C
 *   value           DEVICE [NB][NS][NB][2] fp32 expected accepted progress
 *                   V_B(s, z): value[b][k][j][f] for candidate b, s bin k,
 *                   previous block size candidate j and full-acceptance flag f
 * Unsorted or repeated candidates, or decreasing edges, give RG_ERR_SHAPE;
 * NB or NS out of range RG_ERR_UNSUPPORTED.
 */
typedef struct rg_block_policy {
  int32_t num_candidates;
  const int32_t* candidates;
  int32_t num_s_bins;
  const float* s_edges;
  const float* cost;
  float rho;
  const float* value;
} rg_block_policy;

/*
 * One round of block sizing for a batch (Sec. 5.2), then the requests grouped
 * by planned size (Sec. 5.3).  Per request r, after the verification of its
 * block of size B_{t-1} = prev_block[r]:
 *
 *   s = -(accept_entropy[r] + entropy_hist[r]) / 2     (Eq. 2: e_{t-1}, e_{t-2})
 *   j = the largest candidate index with candidates[j] <= B_{t-1} (0 if none)
 *   f = 1 if accept_len[r] >= B_{t-1} (the block was accepted in full) else 0
 *   next_block[r] = the candidate B maximising value[B][bin(s)][j][f] -
 *                   rho * cost[B] (Eq. 3), the smaller candidate on ties
 *   entropy_hist[r] = accept_entropy[r]   (the history for the next round)
 *
 * computed in fp32 with one rounding per operation (no fused multiply-add).
 *
 *   accept_len, accept_entropy  DEVICE [R] rg_verify_accept outputs of the
 *                   round just verified (accept_entropy is its e_t)
 *   prev_block      DEVICE [R] size of the block that round verified
 *   entropy_hist    DEVICE [R] in: the entropy of the round before; out: the
 *                   entropy of this round (the caller seeds new requests)
 *   num_requests    R, 0 .. 65536
 *   next_block      DEVICE [R] out: planned block size
 *   order           DEVICE [R] out: request indices grouped by planned block
 *                   size, smaller sizes first, ascending index within a size
 *                   (a stable sort); may be NULL when R = 0
 *   bucket_offsets  DEVICE [NB+1] out: candidate b's requests are
 *                   order[bucket_offsets[b] .. bucket_offsets[b+1]-1];
 *                   NULL (with order NULL) to skip the grouping
 * One launch of one work group; no workspace.
 */
rg_status rg_plan_block_sizes(const rg_block_policy* policy, const int32_t* accept_len,
                              const float* accept_entropy, const int32_t* prev_block, float* entropy_hist,
                              int32_t num_requests, int32_t* next_block, int32_t* order,
                              int32_t* bucket_offsets, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* RECGUIDE_H */
