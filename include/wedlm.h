/*
 * wedlm.h -- C ABI of the WeDLM streaming parallel-decode step on MI355X
 * (gfx950).  WeDLM: arXiv 2512.22737.
 *
 * One decode step of Algorithm 1 (Streaming Parallel Decoding) for a batch of
 * B independent sequences is four calls, in this order, on one stream:
 *
 *   wedlm_reorder      topological reordering of the W-slot window (Eq. 5/6)
 *                      and RoPE at logical positions (Eq. 2)
 *   wedlm_window_attn  causal GQA attention of the reordered window over the
 *                      paged prefix KV cache (Sec. 4.1, Algorithm 1 Forward)
 *   wedlm_score        entropy / greedy token of every mask slot (Sec. 5.2)
 *   wedlm_commit       commit of the leftmost filled run, KV append,
 *                      SelectByEntropy with the adjusted entropy of Eq. (11),
 *                      greedy Sample, refill (Algorithm 1)
 *
 * wedlm_commit_rule is wedlm_commit under a chosen decoding rule: Algorithm
 * 1's streaming rule, block-wise stop-and-wait (Fig. 3, Sec. 6.4) or one
 * token per step (Sec. 6.2).
 *
 * Conventions shared by every call
 * --------------------------------
 *  - All array pointers are DEVICE pointers into memory the caller owns
 *    (contiguous, row-major, naturally aligned; bf16 arrays 16-byte
 *    aligned).  The library never allocates, frees or synchronises: each
 *    call validates its scalar arguments on the host, enqueues its kernels
 *    on `stream` (a hipStream_t; NULL = the default stream) and returns.
 *  - bf16 values are passed as their uint16_t bit patterns.
 *  - Return value: WEDLM_OK (0), or a negative WEDLM_E_* code detected on
 *    the host before anything was enqueued (WEDLM_E_LAUNCH: a launch
 *    failed; kernels enqueued before it may have run).
 *  - Shape limits: 1 <= W <= 64; D in {64, 128}; Hq % Hkv == 0; B >= 1;
 *    16-token pages.
 *  - A mask slot ([M]) is the token id -1; the kernels treat every negative
 *    id as [M].  Logical slot s of sequence b holds logical position
 *    win_start[b] + s (0-based: the committed prefix is positions
 *    0 .. win_start[b]-1).
 *  - Device-side problems that depend on data (a page id outside the cache,
 *    a prefix longer than the block table or than max_prefix_len) never
 *    cause an out-of-bounds access: the affected sequence's status word gets
 *    a WEDLM_SEQ_* bit and its outputs for that call are left unspecified
 *    (wedlm_commit then changes nothing for that sequence).
 *
 * Cache layout (ours; chosen so that both MFMA operands of the attention
 * stream straight from the pages):
 *    k_cache  [num_pages, Hkv, 16, D]   key rows of a page, token-major
 *    v_cache  [num_pages, Hkv, D, 16]   value rows of a page, transposed
 *    block_table [B, max_pages] int32   page id of each 16-position block
 *    position p of sequence b lives in page block_table[b][p / 16], row
 *    p % 16; its "slot" is block_table[b][p / 16] * 16 + p % 16.
 */
#ifndef WEDLM_H
#define WEDLM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define WEDLM_MASK_TOKEN (-1)
#define WEDLM_PAGE_SIZE 16
#define WEDLM_MAX_WINDOW 64

enum {
  WEDLM_OK = 0,
  WEDLM_E_ARG = -1,       /* NULL pointer or bad scalar (tau, T, theta ...) */
  WEDLM_E_SHAPE = -2,     /* unsupported or inconsistent shape              */
  WEDLM_E_WORKSPACE = -3, /* workspace smaller than the *_workspace_size()  */
  WEDLM_E_LAUNCH = -4,    /* a kernel launch failed                         */
  WEDLM_E_DEVICE = -5,    /* no usable gfx950 device                        */
  WEDLM_E_SCRATCH = -6    /* needs more than the library's fixed scratch    */
};

/* per-sequence status bits (int32 status[B]); 0 = fine */
#define WEDLM_SEQ_CAPACITY 1 /* a needed position has no page (table full)  */
#define WEDLM_SEQ_BAD_PAGE 2 /* a block-table entry is outside the cache    */
#define WEDLM_SEQ_BAD_LEN 4  /* prefix length < 0 or > max_prefix_len      */

/* decoding rules of wedlm_commit_rule */
#define WEDLM_RULE_STREAMING 0 /* Algorithm 1 (what wedlm_commit does)     */
#define WEDLM_RULE_BLOCK 1     /* block-wise stop-and-wait commit          */
#define WEDLM_RULE_ONE_TOKEN 2 /* one mask filled per step                 */

/*
 * wedlm_reorder -- Topological reordering, Eq. (5) and Eq. (6), plus the
 * decoupled positional representation of Eq. (2) (RoPE at logical
 * positions), Sec. 4.1 and Algorithm 1's reorder step.
 *
 * Per sequence b, the window's filled slots move to the physical front in
 * ascending logical order, the mask slots follow in ascending logical order
 * (a stable partition; the result is unique).  Physical row i takes logical
 * slot perm[b][i] with logical position pos_ids[b][i] = win_start[b] +
 * perm[b][i].
 *
 * In:
 *   win_tok   [B, W] int32    window tokens, logical slot order (-1 = [M])
 *   win_start [B] int32       committed prefix length c of each sequence
 *   qkv_in    [B, W, Hq+2*Hkv, D] bf16  per slot, logical order: Hq query
 *             heads, then Hkv key heads, then Hkv value heads, pre-RoPE
 *   rope_theta  RoPE base (> 1).  Dimension i pairs with i + D/2 ("rotate
 *             half") at angle pos * rope_theta^(-2i/D); angles and the
 *             rotation are computed in fp64, results rounded to bf16.
 * Out:
 *   perm      [B, W] int32    logical slot of each physical row
 *   pos_ids   [B, W] int32    logical position of each physical row
 *   tok_phys  [B, W] int32    token of each physical row (-1 = [M])
 *   n_obs     [B] int32       number of filled slots
 *   q_phys    [B, W, Hq, D] bf16   rotated queries, physical order
 *   k_phys    [B, W, Hkv, D] bf16  rotated keys, physical order
 *   v_phys    [B, W, Hkv, D] bf16  values, physical order (copied)
 * qkv_in, q_phys, k_phys and v_phys may all be NULL: the call then writes
 * perm, pos_ids, tok_phys and n_obs only (a decoder computes its own
 * queries and keys in physical order); some but not all NULL is
 * WEDLM_E_ARG.
 */
int wedlm_reorder(const int32_t* win_tok, const int32_t* win_start,
                  const uint16_t* qkv_in, int32_t B, int32_t W, int32_t Hq,
                  int32_t Hkv, int32_t D, double rope_theta, int32_t* perm,
                  int32_t* pos_ids, int32_t* tok_phys, int32_t* n_obs,
                  uint16_t* q_phys, uint16_t* k_phys, uint16_t* v_phys,
                  void* stream);

/*
 * wedlm_window_attn -- the attention of Algorithm 1's Forward on the
 * reordered window (Sec. 4.1 "Context Awareness under Causal Masking";
 * Sec. 5.2 "Immediate Caching under Standard Causal Attention").
 *
 * For sequence b, physical row i and query head h (kv head h / (Hq/Hkv)):
 *   out[b][i][h] = softmax_k(q . k_k * softmax_scale) . v_k over the keys
 *   {cached prefix positions 0 .. prefix_len[b]-1} and {window physical
 *   rows 0 .. i} (a plain causal mask with the diagonal; the reordering has
 *   already put every filled slot before every mask).  Window keys/values
 *   come from k_phys / v_phys, the prefix from the paged cache.
 *
 * In:
 *   q_phys, k_phys, v_phys   outputs of wedlm_reorder
 *   k_cache, v_cache         paged cache (layout above), num_pages pages
 *   block_table [B, max_pages], prefix_len [B] (= win_start)
 *   max_prefix_len  an upper bound of every prefix_len[b]; it sizes the
 *                   split of the prefix and the workspace
 *   softmax_scale   usually 1/sqrt(D)
 * Out:
 *   out  [B, W, Hq, D] bf16
 *   lse  [B, W, Hq] fp32 natural-log softmax normaliser, or NULL
 *   status [B] int32 (may be NULL): WEDLM_SEQ_* bits are OR-ed in
 * Workspace: at least wedlm_window_attn_workspace_size(...) bytes of device
 *   memory, 256-byte aligned, contents irrelevant; calls that share one
 *   workspace must not overlap.
 */
size_t wedlm_window_attn_workspace_size(int32_t B, int32_t W, int32_t Hq,
                                        int32_t Hkv, int32_t D,
                                        int32_t max_prefix_len);
int wedlm_window_attn(const uint16_t* q_phys, const uint16_t* k_phys,
                      const uint16_t* v_phys, const uint16_t* k_cache,
                      const uint16_t* v_cache, int64_t num_pages,
                      const int32_t* block_table, int32_t max_pages,
                      const int32_t* prefix_len, int32_t B, int32_t W,
                      int32_t Hq, int32_t Hkv, int32_t D,
                      int32_t max_prefix_len, float softmax_scale,
                      uint16_t* out, float* lse, int32_t* status,
                      void* workspace, size_t workspace_bytes, void* stream);

/*
 * wedlm_window_attn_noalloc -- wedlm_window_attn for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  Same arguments, operation,
 * layouts and results as wedlm_window_attn, without the workspace: the
 * split-K partials go to a scratch array of WEDLM_ATTN_SCRATCH_BYTES that
 * the library holds in each device's memory from load to process exit.
 * Nothing is allocated or freed by the call.
 *
 * Limit: the call's workspace need, wedlm_window_attn_workspace_size(B, W,
 * Hq, Hkv, D, max_prefix_len), must not exceed WEDLM_ATTN_SCRATCH_BYTES
 * (64 MiB: e.g. 8 sequences x 8 kv heads x 256 query rows over 4 splits at
 * D = 128 need 34 MiB); otherwise WEDLM_E_SCRATCH and nothing is enqueued.
 * Every call on a GPU shares that GPU's array, which keeps the last call's
 * contents (nothing in it needs to start at zero): calls that overlap on
 * one GPU (other streams, other threads) race and must be serialised by the
 * caller.  WEDLM_E_DEVICE if the array's device address cannot be obtained.
 */
#define WEDLM_ATTN_SCRATCH_BYTES ((size_t)64 << 20)
int wedlm_window_attn_noalloc(const uint16_t* q_phys, const uint16_t* k_phys,
                              const uint16_t* v_phys, const uint16_t* k_cache,
                              const uint16_t* v_cache, int64_t num_pages,
                              const int32_t* block_table, int32_t max_pages,
                              const int32_t* prefix_len, int32_t B, int32_t W,
                              int32_t Hq, int32_t Hkv, int32_t D,
                              int32_t max_prefix_len, float softmax_scale,
                              uint16_t* out, float* lse, int32_t* status,
                              void* stream);

/*
 * wedlm_score -- per mask slot, the greedy token and the entropy of the
 * predicted distribution (Sec. 5.2, the H_i inside Eq. (11)).
 *
 * For every masked physical row i >= n_obs[b] (rows below are not read):
 *   argmax[b][i]  = lowest token id among the maximal raw fp32 logits
 *   entropy[b][i] = H = -sum_v p_v ln p_v, p = softmax(logits / temperature)
 *                   (nats), computed as ln(1+R) + S/(1+R) with
 *                   R = sum_{v != argmax} e^{z_v}, S = sum_{v != argmax}
 *                   -z_v e^{z_v}, z_v = (l_v - l_max)/T, accumulated in fp64
 *   pmax[b][i]    = 1 / (1 + R), the top probability
 * Entries of observed rows are left untouched.
 *
 * In:
 *   logits [B, W, V] fp32, physical row order; row (b, i) starts at
 *          logits + (b*W + i) * row_stride (row_stride >= V, in elements;
 *          rows on 16-byte boundaries stream faster).  Values must be
 *          finite or -inf.
 *   n_obs  [B] int32 (from wedlm_reorder)
 *   temperature  > 0
 * Out: argmax [B, W] int32, entropy [B, W] fp32, pmax [B, W] fp32 (may be
 *   NULL).
 * Workspace: wedlm_score_workspace_size(B, W, V) bytes (may be 0 with a
 *   NULL workspace when that size is 0).
 */
size_t wedlm_score_workspace_size(int32_t B, int32_t W, int32_t V);
int wedlm_score(const float* logits, int64_t row_stride, const int32_t* n_obs,
                int32_t B, int32_t W, int32_t V, double temperature,
                int32_t* argmax, float* entropy, float* pmax, void* workspace,
                size_t workspace_bytes, void* stream);

/*
 * wedlm_commit -- Algorithm 1 after the forward: commit, KV extend,
 * SelectByEntropy (Eq. 11), Sample, refill.  In place on the window state.
 *
 * Per sequence b with c = win_start[b]:
 *  1. n = length of the leading run of filled slots in logical order.
 *     Those tokens are committed: committed_tok[b][j] = win_tok[b][j],
 *     committed_slot[b][j] = slot of position c + j (j < n; -1 after).
 *     They are exactly physical rows 0..n-1, whose rotated K and V rows
 *     (k_phys / v_phys) are copied into the cache at those slots.
 *  2. For every mask slot s, with s0 the leftmost mask and d = s - s0,
 *     H = entropy of s's physical row: s is selected iff
 *     (double)H < tau - lambda * d  (fp64, no fused multiply-add).
 *     If no mask passes and at least one exists, the single mask with the
 *     smallest (double)H + lambda * d is selected (ties: leftmost), the
 *     lowest-entropy one-token rule of Sec. 6.2.
 *  3. Each selected mask takes argmax of its physical row (greedy Sample).
 *  4. The window drops its first n slots and appends n masks; win_start
 *     advances by n.
 *  selected[b][s] (logical slots, before the shift): 1 = passed the
 *  threshold, 2 = fallback, 0 = not selected.
 *
 * In/out: win_tok [B, W], win_start [B], k_cache, v_cache.
 * In:  argmax, entropy [B, W] (wedlm_score), k_phys, v_phys
 *      (wedlm_reorder), block_table [B, max_pages], num_pages.
 * Out: n_commit [B], committed_tok [B, W], committed_slot [B, W],
 *      selected [B, W] uint8, status [B] (set, not OR-ed: 0 or WEDLM_SEQ_*).
 *      If any committed position lacks a valid page, that sequence's state
 *      is left unchanged, n_commit = 0 and status says why.
 */
int wedlm_commit(int32_t* win_tok, int32_t* win_start, const int32_t* argmax,
                 const float* entropy, double tau, double lambda,
                 const uint16_t* k_phys, const uint16_t* v_phys,
                 uint16_t* k_cache, uint16_t* v_cache, int64_t num_pages,
                 const int32_t* block_table, int32_t max_pages, int32_t B,
                 int32_t W, int32_t Hkv, int32_t D, int32_t* n_commit,
                 int32_t* committed_tok, int32_t* committed_slot,
                 uint8_t* selected, int32_t* status, void* stream);

/*
 * wedlm_commit_rule -- wedlm_commit under the decoding rule `rule`, for
 * comparing Algorithm 1 with the rules the paper measures it against.
 * Arguments, layouts, outputs and errors are those of wedlm_commit; `rule`
 * changes steps 1 and 2 only:
 *   WEDLM_RULE_STREAMING  exactly wedlm_commit (Algorithm 1).
 *   WEDLM_RULE_BLOCK      block-wise decoding with stop-and-wait commit
 *                         (Fig. 3; Sec. 6.4 and Fig. 4c): the block is the
 *                         W-slot window.  n = W if no slot is a mask, else
 *                         n = 0, so nothing is committed until the whole
 *                         block is filled; then all W slots commit and the
 *                         window refills with W masks.  Selection as in
 *                         step 2 (d measured from the leftmost mask).
 *   WEDLM_RULE_ONE_TOKEN  the unified step-wise scheme of Sec. 6.2: exactly
 *                         one mask per step, the one with the smallest
 *                         (double)H + lambda * d (ties: leftmost), whatever
 *                         tau; selected = 2 for it.  Commit as in step 1.
 * Any other rule value returns WEDLM_E_ARG.
 */
int wedlm_commit_rule(int32_t* win_tok, int32_t* win_start,
                      const int32_t* argmax, const float* entropy, double tau,
                      double lambda, const uint16_t* k_phys,
                      const uint16_t* v_phys, uint16_t* k_cache,
                      uint16_t* v_cache, int64_t num_pages,
                      const int32_t* block_table, int32_t max_pages, int32_t B,
                      int32_t W, int32_t Hkv, int32_t D, int32_t* n_commit,
                      int32_t* committed_tok, int32_t* committed_slot,
                      uint8_t* selected, int32_t* status, int32_t rule,
                      void* stream);

/*
 * wedlm_lm_head_score -- the output layer of the window forward fused with
 * the score of its rows: the logits that the mask slots are scored on
 * (Algorithm 1's Forward and SelectByEntropy; the H_i of Eq. (11),
 * Sec. 5.2), reduced to the greedy token, entropy and top probability
 * without writing the logits to memory.
 *
 * For each row r:  logits[v] = sum_k hidden[r][k] * w_vocab[v][k] (bf16
 * products, fp32 accumulation on MFMA), then with p = softmax(logits / T):
 *   argmax[r]  = the first v holding the largest logit (fp32)
 *   entropy[r] = -sum_v p_v ln p_v (nats), pmax[r] = max_v p_v
 *
 * In:
 *   hidden   [R, Hd] bf16   rows to score (e.g. the final hidden states of
 *                           the window's mask rows), row-major
 *   w_vocab  [V, Hd] bf16   output-layer weight, one row per token
 *   Hd a multiple of 256; R, V >= 1; temperature > 0
 * Out:
 *   argmax [R] int32, entropy [R] fp32, pmax [R] fp32 or NULL
 * Workspace: wedlm_lm_head_score_workspace_size(R, Hd, V) bytes (0 when the
 *   vocabulary fits one tile); per-tile partial states, contents undefined.
 * Errors: WEDLM_E_ARG (NULL pointer, temperature), WEDLM_E_SHAPE,
 *   WEDLM_E_WORKSPACE, WEDLM_E_LAUNCH.
 */
size_t wedlm_lm_head_score_workspace_size(int32_t R, int32_t Hd, int32_t V);
int wedlm_lm_head_score(const uint16_t* hidden, const uint16_t* w_vocab,
                        int32_t R, int32_t Hd, int32_t V, double temperature,
                        int32_t* argmax, float* entropy, float* pmax,
                        void* workspace, size_t workspace_bytes,
                        void* stream);

/* Message for a WEDLM_* return code (static storage). */
const char* wedlm_strerror(int code);

/* Library version, major * 10000 + minor * 100 + patch. */
int wedlm_version(void);

#ifdef __cplusplus
}
#endif

#endif /* WEDLM_H */
