/*
 * echo.h -- C ABI of the batch super-tree verification library (MI355X / gfx950).
 *
 * One speculative-decoding step of a batch of R requests verifies a single
 * "super-tree": the union of every request's draft candidates, under one
 * batch-wide verification budget (the cap sum_i K_i <= K_max of eq. 4).  The
 * four calls below are the four stages of that step:
 *
 *   echo_gate             path scores (eq. 5) and the global top-B selection
 *   echo_build_tree_mask  flatten & pack of the selection (Fig. 3, stage 3)
 *   echo_tree_verify_attn tree-masked GQA attention of every verify slot
 *                         (the single verification forward, Section 3.1)
 *   echo_accept           greedy acceptance of the longest matching path
 *
 * Conventions shared by every call
 * --------------------------------
 * - Every array argument is a DEVICE pointer owned by the caller.  The
 *   library never allocates device memory: scratch space is the caller's
 *   `workspace` (size from the matching *_workspace_size call, any
 *   256-byte-aligned device buffer; contents on entry are ignored).
 * - Every call is asynchronous on `stream` (a hipStream_t; NULL = the null
 *   stream), performs no host synchronisation and may be captured in a HIP
 *   graph.  Calls on one stream run in order; the same workspace must not be
 *   used by two calls that may run concurrently.
 * - Return value: ECHO_OK, or a negative host-detected error, in which case
 *   nothing was enqueued.
 * - `status` (nullable device int32) receives the OR of ECHO_DATA_* bits for
 *   problems found in the data itself.  The library ORs into it and never
 *   clears it.  Data problems never abort: each is clamped as documented and
 *   all outputs are still written.
 * - Outputs sized by a capacity (R + budget verify slots) are written only
 *   for the rows that exist (q_offsets[R]); later rows are left untouched.
 * - bfloat16 tensors are passed as uint16_t bit patterns.
 */
#ifndef ECHO_H
#define ECHO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef void* echo_stream_t; /* hipStream_t */

/* ---- return codes ------------------------------------------------------ */
#define ECHO_OK 0
#define ECHO_ERR_INVALID_ARG (-1) /* null pointer, negative or inconsistent size  */
#define ECHO_ERR_UNSUPPORTED (-2) /* head_dim != 128, limits below exceeded       */
#define ECHO_ERR_WORKSPACE (-3)   /* workspace too small or misaligned            */
#define ECHO_ERR_HIP (-4)         /* a HIP runtime call or kernel launch failed   */

/* ---- data-error bits OR-ed into *status -------------------------------- */
#define ECHO_DATA_NAN_LOGQ (1 << 0)        /* NaN log q: treated as -inf                    */
#define ECHO_DATA_POS_LOGQ (1 << 1)        /* log q > 0: treated as 0                       */
#define ECHO_DATA_BAD_PARENT (1 << 2)      /* parent not in [-1, local index): treated as -1 */
#define ECHO_DATA_TOO_DEEP (1 << 3)        /* depth > ECHO_MAX_DEPTH: path score -inf       */
#define ECHO_DATA_NOT_CLOSED (1 << 4)      /* selected node whose parent is not selected    */
#define ECHO_DATA_OVER_CAPACITY (1 << 5)   /* more selected nodes than budget               */
#define ECHO_DATA_BAD_SLOT_PARENT (1 << 6) /* slot_parent not in [0, slot)                  */
#define ECHO_DATA_BAD_OFFSETS (1 << 7)     /* decreasing / out-of-capacity offsets          */

/* ---- limits ------------------------------------------------------------ */
#define ECHO_MAX_DEPTH 16       /* deepest draft node that can be selected           */
#define ECHO_HEAD_DIM 128       /* the only supported head dimension                 */
#define ECHO_MAX_BUDGET 16384   /* largest budget B                                  */
#define ECHO_MAX_REQUESTS 4095  /* largest batch R                                   */
#define ECHO_MAX_CHECKPOINTS 16 /* entries of a sparse-gating checkpoint table       */

/*
 * echo_gate -- path scores and the global top-B selection.
 *
 * Path score (eq. 5): S_j = S_pa(j) + log q_j, S = 0 at the root, folded from
 * the root towards the leaf with one IEEE binary32 add per level.  Selection
 * (eq. 4 budget; Theorem 2 / Proposition 1 exchange argument): the
 * min(budget, #finite S) candidates of the whole batch with the largest S;
 * ties go to the smaller global candidate index; S = -inf is never selected.
 * Because log q <= 0 (after the clamps below) a parent's S is at least its
 * child's and its index is smaller, so the selection is closed under parents
 * by construction; this call never sets ECHO_DATA_NOT_CLOSED.
 *
 *   cand_offsets [R+1] int32   request-major CSR of candidates; g = cand_offsets[r] + n
 *   parent       [N]   int32   request-local parent index, -1 = child of the root;
 *                              must be < n (parents precede children)
 *   logq         [N]   float   draft log-probability of the candidate token
 *   budget                     B >= 0 draft nodes (<= ECHO_MAX_BUDGET)
 *   path_score   [N]   float   (nullable) S per candidate after the clamps
 *   selected     [N]   uint8   1 = verified this step, 0 = not
 *   num_selected [1]   int32   min(budget, #finite S)
 * Clamps: NaN log q -> -inf; log q > 0 -> 0; bad parent -> -1; depth >
 * ECHO_MAX_DEPTH -> S = -inf.  N must equal cand_offsets[R] (not checked on
 * the host: the offsets are device data).
 */
int32_t echo_gate(const int32_t* cand_offsets, const int32_t* parent, const float* logq,
                  int32_t R, int32_t N, int32_t budget, float* path_score, uint8_t* selected,
                  int32_t* num_selected, void* workspace, size_t workspace_bytes, int32_t* status,
                  echo_stream_t stream);
size_t echo_gate_workspace_size(int32_t R, int32_t N, int32_t budget);

/*
 * echo_gate_noalloc -- echo_gate without a caller workspace, for callers that
 * cannot allocate device memory (work under graph capture, serving loops and
 * harnesses that forbid hipMalloc).  It allocates nothing: the workspace is a
 * fixed ECHO_GATE_SCRATCH_BYTES array of the library, one copy per device,
 * held from the first call on a device until the process ends; the caller
 * still passes every input and output.  Arguments, outputs, clamps and status
 * bits are echo_gate's.  Sizes whose workspace exceeds the array
 * (echo_gate_workspace_size(R, N, budget) > ECHO_GATE_SCRATCH_BYTES; every
 * N <= 262144 fits at any R <= ECHO_MAX_REQUESTS) give ECHO_ERR_UNSUPPORTED
 * before any runtime call.  Calls on one device share the array, so calls
 * that overlap on one device (different streams or threads) race and give
 * undefined selections; serialise them.  The first call on a device looks the
 * array's device address up (ECHO_ERR_HIP if that fails).
 */
#define ECHO_GATE_SCRATCH_BYTES (8u << 20)
int32_t echo_gate_noalloc(const int32_t* cand_offsets, const int32_t* parent, const float* logq,
                          int32_t R, int32_t N, int32_t budget, float* path_score,
                          uint8_t* selected, int32_t* num_selected, int32_t* status,
                          echo_stream_t stream);

/*
 * echo_gate_sparse -- echo_gate preceded by sparse gating at checkpoint depths
 * (Section 3.2: layer confidence eq. 6, gating signal eq. 7; truncation as in
 * phase 1 of Alg. 1).
 *
 * For every request r and checkpoint depth d the layer confidence is the
 * largest path score among r's depth-d candidates (eq. 6 without the exp;
 * -inf if there is none).  Request r passes the checkpoint iff that maximum is
 * strictly greater than ln tau_d (eq. 7 in the log domain, compared in
 * binary32).  At the first checkpoint depth t_r it fails, the request is
 * truncated: none of its candidates at depth >= t_r can be selected.  The
 * global top-B of echo_gate then runs over the candidates that remain, so the
 * budget a truncated request frees goes to the other requests' depth or to
 * this request's width above t_r.
 *
 *   sig_depth    [num_sig] int32  HOST array: checkpoint depths, 1..ECHO_MAX_DEPTH
 *                                 (1 = the root's children); a depth listed twice
 *                                 must pass both thresholds
 *   log_tau      [num_sig] float  HOST array: ln tau of each checkpoint; -inf
 *                                 passes any depth with a finite score, +inf or
 *                                 0 passes none (scores are <= 0); NaN is refused
 *   num_sig                       0..ECHO_MAX_CHECKPOINTS (0: no truncation)
 *   trunc_depth  [R]       int32  (nullable) t_r, ECHO_MAX_DEPTH + 1 if none fails
 * The checkpoint table is read on the host during the call and travels in the
 * kernel arguments (a captured graph keeps the values of capture time).  All
 * other arguments, outputs, clamps and status bits are those of echo_gate;
 * path_score holds the untruncated eq. 5 scores.  The workspace is that of
 * echo_gate (echo_gate_sparse_workspace_size returns the same size).
 */
int32_t echo_gate_sparse(const int32_t* cand_offsets, const int32_t* parent, const float* logq,
                         int32_t R, int32_t N, int32_t budget, const int32_t* sig_depth,
                         const float* log_tau, int32_t num_sig, float* path_score,
                         uint8_t* selected, int32_t* num_selected, int32_t* trunc_depth,
                         void* workspace, size_t workspace_bytes, int32_t* status,
                         echo_stream_t stream);
size_t echo_gate_sparse_workspace_size(int32_t R, int32_t N, int32_t budget);

/*
 * echo_gate_elastic -- the selection made by the unified elastic budget
 * scheduler of Alg. 1 (Section 3.3), applied to the drafted candidate pool.
 *
 * Phase 1 (global depth extension, priority 1) walks the depths d = 1, 2, ...
 * while budget is left and some request is active; at each depth the active
 * requests are served in request order.  A request's appendable depth-d
 * candidates are those with a finite path score whose parent it already holds
 * (the root at depth 1).  At a checkpoint depth it passes iff the largest
 * appendable path score is strictly above ln tau_d (eq. 6 and eq. 7 in the log
 * domain; no appendable candidate fails); other depths always pass.  A request
 * that passes takes its min(w_topk, budget left, #appendable) best appendable
 * candidates (path score descending, index ascending) and is charged that
 * many; with none appendable it leaves the active set (its drafted tree is
 * exhausted).  A request that fails is truncated at d and leaves the active
 * set.  Phase 2 (opportunistic width expansion, priority 2) serves the
 * truncated requests in request order while budget is left: a request
 * truncated at depth t >= 2 adds its next best appendable depth-(t-1)
 * candidates, min(budget left, w_max - its width there, #remaining), and is
 * charged that many.  The selection is ancestor-closed by construction.
 *
 *   sig_depth, log_tau, num_sig   HOST checkpoint table, as for echo_gate_sparse
 *   w_topk                        default width per depth, >= 1
 *   w_max                         width a truncated request may widen to, >= 0
 *   num_selected [1]    int32     number of selected candidates (<= budget)
 *   trunc_depth  [R]    int32     (nullable) depth at which the request was
 *                                 truncated in phase 1, ECHO_MAX_DEPTH + 1 if it
 *                                 never was (including requests the budget ran
 *                                 out before testing)
 * Other arguments, clamps and status bits are those of echo_gate.  The
 * workspace is larger than echo_gate's: echo_gate_elastic_workspace_size.
 */
int32_t echo_gate_elastic(const int32_t* cand_offsets, const int32_t* parent, const float* logq,
                          int32_t R, int32_t N, int32_t budget, const int32_t* sig_depth,
                          const float* log_tau, int32_t num_sig, int32_t w_topk, int32_t w_max,
                          float* path_score, uint8_t* selected, int32_t* num_selected,
                          int32_t* trunc_depth, void* workspace, size_t workspace_bytes,
                          int32_t* status, echo_stream_t stream);
size_t echo_gate_elastic_workspace_size(int32_t R, int32_t N, int32_t budget);

/*
 * echo_build_tree_mask -- flatten & pack the selection into verify slots
 * (Fig. 3, stage 3; the paper gives no layout, this is the library's).
 *
 * Request r owns slots [q_offsets[r], q_offsets[r+1]).  Local slot 0 is the
 * root (the last verified token); local slots 1.. are the request's selected
 * candidates in ascending global index, so a parent precedes its children.
 *   q_offsets    [R+1]         int32  exclusive scan of 1 + #selected per request
 *   slot_cand    [R+budget]    int32  global candidate index, -1 for a root
 *   slot_parent  [R+budget]    int32  request-local parent slot, -1 for a root
 *   slot_token   [R+budget]    int32  token[cand] or root_token[r]
 *   position_ids [R+budget]    int32  prefix_len[r] + depth (root depth 0)
 *   tree_mask    [R+budget][mask_words] uint32: bit j (word j>>5, bit j&31)
 *                of row s is set iff local slot j is s or an ancestor of s
 * mask_words must be >= ceil((budget+1)/32).  If more than `budget` nodes
 * are selected only the first `budget` (ascending index) are packed
 * (ECHO_DATA_OVER_CAPACITY).  A selected node whose parent is not selected
 * hangs from its nearest selected ancestor (ECHO_DATA_NOT_CLOSED).
 */
int32_t echo_build_tree_mask(const int32_t* cand_offsets, const int32_t* parent,
                             const int32_t* token, const uint8_t* selected,
                             const int32_t* root_token, const int32_t* prefix_len, int32_t R,
                             int32_t N, int32_t budget, int32_t* q_offsets, int32_t* slot_cand,
                             int32_t* slot_parent, int32_t* slot_token, int32_t* position_ids,
                             uint32_t* tree_mask, int32_t mask_words, void* workspace,
                             size_t workspace_bytes, int32_t* status, echo_stream_t stream);
size_t echo_build_tree_mask_workspace_size(int32_t R, int32_t N, int32_t budget);

/*
 * echo_tree_verify_attn -- tree-masked grouped-query verification attention
 * (the one parallel target forward over the flattened union, Section 3.1;
 * the paper's "specialized operators for irregular batch shapes").
 *
 * Slot s of request r, query head h, uses key/value head h / (Hq/Hkv) and
 * sees the request's KV prefix rows [kv_offsets[r], kv_offsets[r+1]) plus
 * the new keys of its local slots j whose tree_mask bit is set.  Logits
 * sm_scale * <q, k> in fp32, softmax, output sum p * v accumulated in fp32
 * with each probability p rounded to bf16 for the product and the output
 * divided by the sum of the weights used (an exact convex combination of V
 * rows).  Where one key of a 32-key tile may carry more than 1/16 of a row's
 * weight so far, the bf16 residual p - bf16(p) enters a second product, so
 * that rows whose weight sits on a few keys keep 2^-17 of relative error on
 * those weights; elsewhere each weight is within 2^-9 of itself.  A row whose
 * keys are split between workgroups is merged from partial outputs stored in
 * fp16 with a power-of-two scale per row (rounding: 2^-12 of the row's largest
 * partial value).  The LSE uses the fp32 sum.  NaN inputs give unspecified
 * outputs.
 *   q        [max_rows][Hq][128]  bf16 (slot-indexed, RoPE already applied)
 *   k_new, v_new [max_rows][Hkv][128] bf16 (K/V of the verify slots)
 *   k_cache, v_cache [kv_rows][Hkv][128] bf16, token-major (request r's prefix
 *                                 is rows [kv_offsets[r], kv_offsets[r+1]))
 *   kv_offsets [R+1] int64, q_offsets [R+1] int32, tree_mask as above
 *   out      [max_rows][Hq][128]  float
 *   lse      [max_rows][Hq]       float (nullable), natural log; -inf with out = 0
 *                                 for a row that sees no key
 *   sm_scale                      finite and > 0 (else ECHO_ERR_INVALID_ARG): the
 *                                 softmax takes each row's largest raw logit as
 *                                 its reference before scaling
 * Requests with decreasing offsets, q_offsets beyond max_rows or kv_offsets
 * outside [0, kv_rows] are skipped (ECHO_DATA_BAD_OFFSETS); their rows are
 * not written.  Deterministic: no floating-point atomics.
 */
int32_t echo_tree_verify_attn(const uint16_t* q, const uint16_t* k_new, const uint16_t* v_new,
                              const uint16_t* k_cache, const uint16_t* v_cache,
                              const int64_t* kv_offsets, int64_t kv_rows, const int32_t* q_offsets,
                              const uint32_t* tree_mask, int32_t mask_words, int32_t R,
                              int32_t max_rows, int32_t num_q_heads, int32_t num_kv_heads,
                              int32_t head_dim, float sm_scale, float* out, float* lse,
                              void* workspace, size_t workspace_bytes, int32_t* status,
                              echo_stream_t stream);
size_t echo_tree_verify_attn_workspace_size(int32_t R, int32_t max_rows, int32_t num_q_heads,
                                            int32_t num_kv_heads, int32_t head_dim);

/*
 * echo_tree_verify_attn_paged -- echo_tree_verify_attn with each request's KV
 * prefix in a paged cache (the block-table layout of serving engines; the
 * paper leaves the cache layout to the engine).
 *
 * Position p < prefix_len[r] of request r is row p % page_size of page
 * block_table[r * max_pages_per_request + p / page_size]; a page holds
 * page_size token rows of Hkv * 128 bf16 each.
 *   k_pages, v_pages [num_pages][page_size][Hkv][128] bf16
 *   page_size        power of two, >= 32 (a 32-key tile never straddles pages)
 *   block_table      [R][max_pages_per_request] int32 page ids
 *   prefix_len       [R] int32 cached positions per request
 * A request whose prefix needs a page id outside [0, num_pages) (or a length
 * beyond its block-table row) is skipped with ECHO_DATA_BAD_OFFSETS, like an
 * invalid kv_offsets range.  Everything else is as for echo_tree_verify_attn,
 * including the workspace size (ECHO_ERR_UNSUPPORTED in the unlikely case that
 * R * ceil(max_pages_per_request / 256) page-check flags do not fit in it).
 */
int32_t echo_tree_verify_attn_paged(
    const uint16_t* q, const uint16_t* k_new, const uint16_t* v_new, const uint16_t* k_pages,
    const uint16_t* v_pages, int64_t num_pages, int32_t page_size, const int32_t* block_table,
    int32_t max_pages_per_request, const int32_t* prefix_len, const int32_t* q_offsets,
    const uint32_t* tree_mask, int32_t mask_words, int32_t R, int32_t max_rows,
    int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim, float sm_scale, float* out,
    float* lse, void* workspace, size_t workspace_bytes, int32_t* status, echo_stream_t stream);

/*
 * echo_accept -- greedy acceptance (Section 2 standard SD, greedy decoding).
 *
 * Root slot valid; slot s valid iff its parent is valid, its depth <=
 * max_depth and slot_token[s] == target_token[parent slot].  The path ends at
 * the deepest valid slot (ties: smallest local slot).
 *   target_token [max_rows] int32  target argmax after each slot
 *   accept_len   [R]        int32  depth of the end slot (0..max_depth)
 *   accept_slots [R][max_depth] int32 global slot indices of the accepted
 *                           path from depth 1 to the end slot, -1 padded
 *   bonus_token  [R]        int32  target_token[end slot] (-1 if no slots)
 * max_depth in [1, ECHO_MAX_DEPTH].
 */
int32_t echo_accept(const int32_t* q_offsets, const int32_t* slot_parent,
                    const int32_t* slot_token, const int32_t* target_token, int32_t R,
                    int32_t max_rows, int32_t max_depth, int32_t* accept_len,
                    int32_t* accept_slots, int32_t* bonus_token, int32_t* status,
                    echo_stream_t stream);

/*
 * echo_verify_step -- the four calls above in one: echo_gate,
 * echo_build_tree_mask, echo_tree_verify_attn (contiguous cache) and
 * echo_accept on one stream, with the same arguments (in that order; the
 * mask's unused workspace is dropped, `token` is the mask's candidate tokens,
 * `max_rows` serves the attention and the acceptance) and bit-identical
 * outputs and status bits.  It runs the gate's last phase, flatten & pack and
 * the attention's plan in one single-workgroup launch (the three are one
 * workgroup each and run back to back), and the acceptance inside the
 * attention's combine launch (it reads nothing the attention writes): five
 * launches instead of eight.  Every check of the four calls runs before
 * anything is launched; a failing check launches nothing.
 * Needs mask_words * 32 >= budget + 1 and the same LDS bound as the mask
 * call (ECHO_ERR_UNSUPPORTED beyond it).
 */
int32_t echo_verify_step(
    const int32_t* cand_offsets, const int32_t* parent, const float* logq, const int32_t* token,
    int32_t R, int32_t N, int32_t budget, float* path_score, uint8_t* selected,
    int32_t* num_selected, void* gate_workspace, size_t gate_workspace_bytes,
    const int32_t* root_token, const int32_t* prefix_len, int32_t* q_offsets, int32_t* slot_cand,
    int32_t* slot_parent, int32_t* slot_token, int32_t* position_ids, uint32_t* tree_mask,
    int32_t mask_words, const uint16_t* q, const uint16_t* k_new, const uint16_t* v_new,
    const uint16_t* k_cache, const uint16_t* v_cache, const int64_t* kv_offsets, int64_t kv_rows,
    int32_t max_rows, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
    float sm_scale, float* out, float* lse, void* attn_workspace, size_t attn_workspace_bytes,
    const int32_t* target_token, int32_t max_depth, int32_t* accept_len, int32_t* accept_slots,
    int32_t* bonus_token, int32_t* status, echo_stream_t stream);

/*
 * echo_accept_logits -- echo_accept with the target tokens taken from the
 * target model's logits: the greedy (temperature 0) token after slot s is the
 * argmax of logits[s][0 .. vocab), compared as floats (-0 == +0), NaN never
 * winning over a number, ties to the smaller token id (a row of NaN gives 0).
 *   logits       [max_rows][vocab] bf16, row-major
 *   target_token [max_rows] int32  OUTPUT: the argmax of every existing row
 * The other arguments and outputs are those of echo_accept.  The argmax reads
 * q_offsets[R] * vocab * 2 bytes: it is bound by HBM bandwidth.
 */
int32_t echo_accept_logits(const int32_t* q_offsets, const int32_t* slot_parent,
                           const int32_t* slot_token, const uint16_t* logits, int64_t vocab,
                           int32_t R, int32_t max_rows, int32_t max_depth, int32_t* target_token,
                           int32_t* accept_len, int32_t* accept_slots, int32_t* bonus_token,
                           int32_t* status, echo_stream_t stream);

/*
 * echo_commit_kv -- append each request's verified root and accepted path to
 * its paged KV cache (the step after acceptance; the paper leaves the cache
 * to the serving engine).
 *
 * For a request with verify slots, rows k_new/v_new[q_offsets[r]] (the root)
 * and k_new/v_new[accept_slots[r][j]], j < accept_len[r], are written at
 * positions prefix_len[r], prefix_len[r] + 1, ... (page layout as for
 * echo_tree_verify_attn_paged), and prefix_len[r] grows by 1 + accept_len[r]
 * (in place).  The caller provides the pages: if a position needs a page id
 * outside [0, num_pages), or a slot index is outside [0, max_rows), nothing
 * of that request is written (ECHO_DATA_BAD_OFFSETS).  Requests without slots
 * are left unchanged.
 *   accept_len [R], accept_slots [R][max_depth]  as written by echo_accept
 *   k_new, v_new [max_rows][Hkv][128] bf16; k_pages, v_pages as above
 *   page_size   any positive size; pointers 16-byte aligned
 */
int32_t echo_commit_kv(const int32_t* q_offsets, const int32_t* accept_len,
                       const int32_t* accept_slots, int32_t max_depth, const uint16_t* k_new,
                       const uint16_t* v_new, int32_t R, int32_t max_rows, int32_t num_kv_heads,
                       uint16_t* k_pages, uint16_t* v_pages, int64_t num_pages, int32_t page_size,
                       const int32_t* block_table, int32_t max_pages_per_request,
                       int32_t* prefix_len, int32_t* status, echo_stream_t stream);

/*
 * echo_tree_verify_attn_timed, echo_tree_verify_attn_paged_timed -- the two
 * attention calls above with a measurement of their main kernel (not a step
 * of the method).  `ev_start` and `ev_stop` (hipEvent_t, both non-null,
 * created by the caller) are recorded on `stream` right before and right
 * after the main attention kernel of this call only, so that a harness can
 * time that kernel alone.  The event packets leave a few microseconds of idle
 * time around the kernel: a step timed for throughput uses the untimed calls.
 * Every other argument, output and error is that of the untimed call; null
 * events give ECHO_ERR_INVALID_ARG.
 */
int32_t echo_tree_verify_attn_timed(const uint16_t* q, const uint16_t* k_new,
                                    const uint16_t* v_new, const uint16_t* k_cache,
                                    const uint16_t* v_cache, const int64_t* kv_offsets,
                                    int64_t kv_rows, const int32_t* q_offsets,
                                    const uint32_t* tree_mask, int32_t mask_words, int32_t R,
                                    int32_t max_rows, int32_t num_q_heads, int32_t num_kv_heads,
                                    int32_t head_dim, float sm_scale, float* out, float* lse,
                                    void* workspace, size_t workspace_bytes, int32_t* status,
                                    void* ev_start, void* ev_stop, echo_stream_t stream);
int32_t echo_tree_verify_attn_paged_timed(
    const uint16_t* q, const uint16_t* k_new, const uint16_t* v_new, const uint16_t* k_pages,
    const uint16_t* v_pages, int64_t num_pages, int32_t page_size, const int32_t* block_table,
    int32_t max_pages_per_request, const int32_t* prefix_len, const int32_t* q_offsets,
    const uint32_t* tree_mask, int32_t mask_words, int32_t R, int32_t max_rows,
    int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim, float sm_scale, float* out,
    float* lse, void* workspace, size_t workspace_bytes, int32_t* status, void* ev_start,
    void* ev_stop, echo_stream_t stream);

/*
 * echo_probe_stream_read -- measurement helper (not a step of the method): the
 * streaming-read ceiling that the verification attention's roofline is read
 * against.  Reads k and v, each [rows][heads][128] bf16 (a token-major KV
 * cache), once and writes nothing but, in the unlikely case that the folded
 * data equals a fixed word, sink[0].
 *   mode 0  plain 16-byte vector loads, one workgroup per CU over contiguous
 *           byte ranges
 *   mode 1  the attention's copy pattern: 32-row tiles, each wave of a
 *           four-wave workgroup copying one head's 256-byte slices of the
 *           tile's rows into LDS with direct-to-LDS loads (heads % 4 == 0,
 *           else ECHO_ERR_UNSUPPORTED; a final partial tile is not read)
 *   mode 2  the same copies with every wave streaming its own contiguous
 *           range of 8 KB blocks (rows * heads % 32 == 0, else
 *           ECHO_ERR_UNSUPPORTED)
 * k, v 16-byte aligned; rows * heads * 256 < 2^40.
 */
int32_t echo_probe_stream_read(const uint16_t* k, const uint16_t* v, int64_t rows, int32_t heads,
                               int32_t mode, uint32_t* sink, echo_stream_t stream);

const char* echo_status_string(int32_t code);
const char* echo_version(void);

#ifdef __cplusplus
}
#endif
#endif /* ECHO_H */
