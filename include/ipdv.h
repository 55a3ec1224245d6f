/*
 * ipdv.h -- C ABI of the verifier-side window scoring library (libipdv.so)
 * for AMD Instinct MI355X (gfx950).
 *
 * The entry points are the verifier's calls in one propose-and-verify
 * step of Interactive-Policy Distillation (Section 3.2.3, "Fused Inference
 * Engine", and Eq. (9)):
 *
 *   verify_attn_paged        -- the verification stage's attention: append the
 *                               proposer's window to the verifier's own paged
 *                               KV cache and score every window row in one
 *                               prefill pass over the resident prefix;
 *   lmhead_logsoftmax_verify -- the verifier's next-token distribution at each
 *                               window row (LM head + log-softmax at
 *                               temperature 1): proposal log-prob, LSE, argmax,
 *                               top-K support (Eq. (5)) and entropy;
 *   accept_scan              -- the verdict stage: the top-K coverage rule of
 *                               Eq. (9) applied as a first-event scan over each
 *                               window, with the EOS and length rules and the
 *                               rollback length shared by both caches;
 *   accept_scan_rule         -- the same scan with the rule variants named
 *                               after Eq. (9) (entropy thresholds, asymmetric
 *                               rules, SKD's fixed one-token handback);
 *   sample_takeover          -- the teacher's replacement token at each
 *                               takeover (Eq. (9), second case), drawn from
 *                               the verifier's distribution at that row;
 *   lmhead_sample            -- the proposer's per-row draw (temperature 1)
 *                               from the same records;
 *   lmhead_pack_w            -- W repacked once into 1 KB blocks (optional
 *                               layout for the calls that read W);
 *   lmhead_logp_gather       -- a model's log-probs at listed vocabulary
 *                               indices (the other model's top-K), which
 *                               complete the union support of Eq. (6);
 *   source_split_kl          -- the per-position values of the source-split
 *                               objective (Eqs. (6), (10), (11)).
 *
 * Conventions common to every entry point:
 *   - All array arguments are DEVICE pointers owned by the caller (except the
 *     host-side shape arguments of the *_workspace_size queries).  The library
 *     allocates no device memory and keeps no state besides a thread-local
 *     error message and the optional thread-local timing hook below.
 *   - Every call only enqueues work on `hip_stream` (a hipStream_t; NULL = the
 *     default stream) and returns; it never synchronises.
 *   - Arrays are dense, row-major, with the shapes given below.  Floating
 *     inputs are IPDV_F32 (float) or IPDV_BF16 (bfloat16) as `dtype` says;
 *     arithmetic accumulates in fp32.
 *   - Return value: IPDV_OK, or a negative ipdv_status when host-side
 *     validation fails (nothing is launched) or a HIP launch fails.
 *     ipdv_last_error() then describes the failure.  Nothing is printed and
 *     nothing aborts.
 *   - Device data that break the documented contract (page ids, lengths that
 *     do not fit the page table) give unspecified outputs; the kernels clamp
 *     every index they read so that no access leaves the caller's buffers.
 *
 * Window convention.  Sequence b has L_b = ctx_lens[b] tokens in this
 * verifier's cache and k_b = cu_q[b+1] - cu_q[b] window rows.  Row i
 * (0 <= i < k_b, batch row cu_q[b] + i) is the token at absolute position
 * L_b + i; its output distribution predicts position L_b + i + 1 and scores
 * proposed token prop_tok[cu_q[b] + i].
 */
#ifndef IPDV_H
#define IPDV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  IPDV_OK = 0,
  IPDV_EINVAL = -1,        /* null required pointer or out-of-range argument  */
  IPDV_EUNSUPPORTED = -2,  /* a shape / dtype combination not implemented      */
  IPDV_EWORKSPACE = -3,    /* workspace null or smaller than the size query    */
  IPDV_EHIP = -4           /* a HIP launch or runtime call failed              */
} ipdv_status;

typedef enum { IPDV_F32 = 0, IPDV_BF16 = 1 } ipdv_dtype;

/* OR'ed into the `dtype` argument of the calls that read the LM-head weight
 * W (lmhead_logsoftmax_verify, sample_takeover, lmhead_sample,
 * lmhead_logp_gather): W is in the tiled layout written by lmhead_pack_w
 * instead of row-major [V, Hd].  bf16 only.  Results are bit-identical to the
 * row-major call; the GEMM's operand loads then read whole cache lines. */
#define IPDV_W_TILED 0x10

/* Driver codes (accept_scan): who proposed the window. */
#define IPDV_DRIVER_S 0   /* the student drives; the teacher verifies */
#define IPDV_DRIVER_T 1   /* the teacher drives; the student verifies */

/* Takeover and handback rules (accept_scan_rule), Section 3.2.1 after
 * Eq. (9): top-K coverage is the paper's rule for both; an entropy threshold
 * may replace either test, and the two may differ.  SKD is coverage takeover
 * with a fixed one-token handback. */
#define IPDV_TAKE_COVERAGE 0   /* take over when the draft is outside the verifier's top-K */
#define IPDV_TAKE_ENTROPY 1    /* take over when ent[row] > tau_take */
#define IPDV_HAND_COVERAGE 0   /* hand back when the draft is inside the verifier's top-K */
#define IPDV_HAND_FIXED_ONE 1  /* the teacher emits one token, then hands back (SKD) */
#define IPDV_HAND_ENTROPY 2    /* hand back when ent[row] <= tau_hand */

/* Distillation support S_t (source_split_kl), Eq. (5) and the text after
 * it; the union is the paper's default (Appendix B.2). */
#define IPDV_SUPPORT_UNION 0
#define IPDV_SUPPORT_STUDENT 1
#define IPDV_SUPPORT_TEACHER 2
#define IPDV_SUPPORT_INTERSECTION 3

/* KL direction per token source (source_split_kl): Eq. (10) is the default;
 * Section 4.3 ablates the other three. */
#define IPDV_LOSS_IPD_SPLIT 0      /* reverse KL where src = S, forward where src = T */
#define IPDV_LOSS_PURE_REVERSE 1
#define IPDV_LOSS_PURE_FORWARD 2
#define IPDV_LOSS_INVERSE_SPLIT 3  /* forward KL where src = S, reverse where src = T */

/* Largest index list per row of lmhead_logp_gather. */
#define IPDV_MAX_GATHER 64

/* Source labels (accept_scan `src`). */
#define IPDV_SRC_S 0
#define IPDV_SRC_T 1
#define IPDV_SRC_DISCARDED 255

/* Largest supported top-K (the paper sweeps K in {4, 8, 16, 32}). */
#define IPDV_MAX_K 32

/*
 * Workspace bytes verify_attn_paged needs for these host-side shape values
 * (0 if the arguments are invalid).  max_q is an upper bound of k_b over the
 * sequences of the call; max_pages_per_seq and page_size as passed to
 * verify_attn_paged.
 */
size_t ipdv_attn_workspace_size(int n_seq, int Hq, int Hkv, int D, int max_q,
                                int max_pages_per_seq, int page_size);

/*
 * verify_attn_paged -- verification-stage attention over the paged cache
 * (Section 3.2.3: the verifier evaluates all unverified drafts of its
 * sub-batch in one prefill pass, computing only the newly appended tokens
 * while the prefix cache stays resident; the proposer's tokens are appended
 * to the verifier's live cache).
 *
 * For every handled sequence b and window row i, in place:
 *   1. append: k_cache/v_cache at position L_b + i  <-  k_new/v_new[cu_q[b]+i];
 *   2. attend: for query head h and KV head g = h / (Hq/Hkv),
 *        out[cu_q[b]+i, h, :] = softmax_j( scale * q[cu_q[b]+i, h, :] . K_j )
 *                               . V_j   over keys j = 0 .. L_b + i (inclusive).
 * Q and K are taken as already position-encoded; no other mask or softcap.
 *
 * q       [T, Hq, D]    window queries (dtype)
 * k_new   [T, Hkv, D]   window keys    (dtype)
 * v_new   [T, Hkv, D]   window values  (dtype)
 * k_cache [num_pages, Hkv, D/32, page_size, 32]
 *                       key pages: per KV head and 32-channel slice, the
 *                       slice of each slot in turn (channel d of a slot at
 *                       [page][g][d/32][slot][d%32]); 16-key MFMA operand
 *                       loads then read whole cache lines (dtype, in/out)
 * v_cache [num_pages, Hkv, D, page_size]   value pages, channel-major: per
 *                                          KV head and channel, one value per
 *                                          slot (dtype, in/out)
 * page_table [B, max_pages_per_seq] int32  pages of sequence b in order;
 *                                          position p lives in page
 *                                          page_table[b][p / page_size], slot
 *                                          p % page_size.  Entries up to
 *                                          (L_b + k_b - 1) / page_size must be
 *                                          valid page ids < num_pages.
 * ctx_lens [B] int32    L_b (>= 0)
 * cu_q    [B+1] int32   window row offsets (non-decreasing, cu_q[0] = 0 for the
 *                       batch; T = cu_q[B])
 * seq_ids [n_seq] int32 the sequences this call handles (the verifier's
 *                       sub-batch, Section 3.2.3 groups requests by verifier);
 *                       NULL = sequences 0 .. n_seq-1.  Rows of other
 *                       sequences are neither read nor written.
 * max_q                 >= k_b for every handled sequence (host-side bound)
 * out     [T, Hq, D]    attention output (dtype)
 * Hq, Hkv, D            Hq % Hkv == 0; D in {64, 128} for bf16, D = 64 for fp32
 * page_size             16, 32 or 64
 * scale                 softmax scale, > 0 (normally 1/sqrt(D))
 * workspace             device buffer of >= ipdv_attn_workspace_size(...)
 *                       bytes (split-KV partial results); contents on entry
 *                       are ignored.
 *
 * Errors: IPDV_EINVAL (null pointer, n_seq < 0, max_q < 1, bad head counts,
 * scale not positive and finite), IPDV_EUNSUPPORTED (D, page_size, dtype),
 * IPDV_EWORKSPACE, IPDV_EHIP.
 */
int verify_attn_paged(const void* q, const void* k_new, const void* v_new,
                      void* k_cache, void* v_cache,
                      const int32_t* page_table, int max_pages_per_seq,
                      const int32_t* ctx_lens, const int32_t* cu_q,
                      const int32_t* seq_ids, int n_seq, int max_q,
                      void* out,
                      int Hq, int Hkv, int D, int page_size, int num_pages, float scale,
                      int dtype, void* workspace, size_t workspace_bytes,
                      void* hip_stream);

/*
 * ipdv_check_page_table -- host-side check of the device-data contract of
 * verify_attn_paged (the kernels clamp every index they read, so a table
 * that breaks the contract gives wrong outputs, not faults).  Takes HOST
 * copies of the call's arrays (page_table [B, max_pages_per_seq], ctx_lens
 * [B], cu_q [B+1], seq_ids [n_seq] or NULL) and checks, for every handled
 * sequence b:
 *   - L_b >= 0 and k_b = cu_q[b+1] - cu_q[b] >= 0, with cu_q[0] = 0 and cu_q
 *     non-decreasing;
 *   - k_b <= max_q, and L_b + k_b <= max_pages_per_seq * page_size;
 *   - every page id that holds a position 0 .. L_b + k_b - 1 lies in
 *     [0, num_pages);
 *   - no page the window writes (positions L_b .. L_b + k_b - 1) is also
 *     visible to another handled sequence (a shared prefix page must be
 *     copied before a sequence appends to it);
 *   - seq_ids entries lie in [0, B) and are distinct.
 * B is the number of rows of page_table / entries of ctx_lens.  Returns
 * IPDV_OK, or IPDV_EINVAL with ipdv_last_error() naming the first violation
 * and *bad_seq (if not NULL) set to its sequence (-1 when none applies).
 * Allocates host memory for the page-ownership map; launches nothing.
 */
int ipdv_check_page_table(const int32_t* page_table, int B, int max_pages_per_seq,
                          const int32_t* ctx_lens, const int32_t* cu_q,
                          const int32_t* seq_ids, int n_seq, int max_q,
                          int page_size, int num_pages, int32_t* bad_seq);

/*
 * verify_attn_paged_noalloc -- verify_attn_paged without a workspace
 * argument, for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation).
 * Same arguments, contract and results as verify_attn_paged (the same
 * kernels and split plan); the split-KV partials go to a scratch array of
 * IPDV_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs on
 * until the process ends.  The call allocates nothing.
 *
 * Limit: calls whose workspace (ipdv_attn_workspace_size) exceeds
 * IPDV_NOALLOC_SCRATCH_BYTES return IPDV_EUNSUPPORTED before launching.
 * Every call on one GPU uses the same scratch: calls that may overlap on one
 * GPU (different streams without ordering, or other threads) race and must
 * be serialised by the caller.  Nothing in the scratch needs to start at
 * zero.
 *
 * Errors: those of verify_attn_paged except IPDV_EWORKSPACE; IPDV_EUNSUPPORTED
 * for a call above the limit.
 */
#define IPDV_NOALLOC_SCRATCH_BYTES (128u << 20)
int verify_attn_paged_noalloc(const void* q, const void* k_new, const void* v_new,
                              void* k_cache, void* v_cache,
                              const int32_t* page_table, int max_pages_per_seq,
                              const int32_t* ctx_lens, const int32_t* cu_q,
                              const int32_t* seq_ids, int n_seq, int max_q,
                              void* out,
                              int Hq, int Hkv, int D, int page_size, int num_pages, float scale,
                              int dtype, void* hip_stream);

/* Workspace bytes lmhead_logsoftmax_verify needs (0 if invalid). */
size_t ipdv_lmhead_workspace_size(int M, int Hd, int V, int K);

/*
 * One query for both workspaces, dispatching to the two typed queries above:
 *   which = IPDV_WS_ATTN:   host_shape_args = {n_seq, Hq, Hkv, D, max_q,
 *                           max_pages_per_seq, page_size}, n = 7;
 *   which = IPDV_WS_LMHEAD: host_shape_args = {M, Hd, V, K}, n = 4.
 * host_shape_args is a HOST array.  Returns 0 for an unknown `which`, a NULL
 * array, a count other than the one listed, or shape values the typed query
 * rejects (ipdv_last_error() then says which).
 */
#define IPDV_WS_ATTN 0
#define IPDV_WS_LMHEAD 1
size_t ipdv_workspace_size(int which, const int32_t* host_shape_args, int n);

/*
 * lmhead_logsoftmax_verify -- the verifier's next-token distribution at each
 * window row (temperature 1, as in the paper's rollouts, Appendix A), without
 * writing the logits to memory.
 *
 * For row m: logits l = hidden[m] . W^T (W is the [V, Hd] nn.Linear /
 * tied-embedding layout), LSE = log sum_v exp(l_v), and
 *   lse[m]        = LSE                                   (fp32)
 *   logp_prop[m]  = l[prop_tok[m]] - LSE  (the log q or log pi term of Eq. (4))
 *   argmax[m]     = the first index of the top-K order
 *   topk_idx[m,:] = Top_K of Eq. (5): the K largest logits, sorted by logit
 *                   descending, lower index first on equal logits
 *   topk_logp[m,:]= l[topk_idx] - LSE
 *   entropy[m]    = -sum_v p_v log p_v  (optional; NULL skips it)
 * Row m's outputs go to row out_rows[m] of each output array when out_rows is
 * non-NULL (scatter into batch-wide arrays), else to row m.
 *
 * hidden  [M, Hd]   (dtype);   W [V, Hd] (dtype);   prop_tok [M] int32 in [0, V)
 * out_rows [M] int32 or NULL
 * lse, logp_prop, entropy: float [rows];  argmax int32 [rows];
 * topk_idx int32 [rows, K];  topk_logp float [rows, K]
 * Requirements: M >= 0, Hd % 64 == 0 and Hd <= 4096, 1 <= V <= 262144,
 * 1 <= K <= min(IPDV_MAX_K, V).
 *
 * Errors: IPDV_EINVAL, IPDV_EUNSUPPORTED (dtype, Hd), IPDV_EWORKSPACE, IPDV_EHIP.
 */
int lmhead_logsoftmax_verify(const void* hidden, const void* W,
                             const int32_t* prop_tok, const int32_t* out_rows,
                             int M, int Hd, int V, int K,
                             float* lse, float* logp_prop, int32_t* argmax,
                             int32_t* topk_idx, float* topk_logp, float* entropy,
                             int dtype, void* workspace, size_t workspace_bytes,
                             void* hip_stream);

/*
 * accept_scan -- the verdict stage (Section 3.2.3) with the top-K coverage
 * rule of Eq. (9), one window per sequence.
 *
 * Row i of sequence b scores draft i = prop_tok[cu_q[b]+i], proposed by the
 * driver; covered_i = the draft appears in topk_idx[cu_q[b]+i, 0..K-1] (the
 * verifier's support).
 *   driver S: drafts are accepted (src S) while covered; the first uncovered
 *     draft is a takeover (rejected; the teacher emits the replacement later;
 *     next driver T).
 *   driver T: drafts are accepted (src T); the first covered draft is a
 *     handback (kept; later drafts discarded; next driver S).
 *   EOS: a student EOS ends the request only if covered (else takeover); a
 *     teacher EOS is accepted and ends it.
 *   length: draft i needs seq_lens[b] + i < max_len; a request whose accepted
 *     drafts reach max_len is finished.
 * Outputs per sequence: n_acc (accepted drafts), event_row (row of the
 * takeover / handback, -1 if none), next_driver, finished (0/1),
 * new_cache_len = L_b + n_acc (+1 after a takeover: the rejected row's input
 * stays cached and the replacement becomes the last token) -- the common
 * boundary both models' caches roll back to; per row: src (IPDV_SRC_*).
 *
 * cu_q [B+1] int32, prop_tok [T] int32, topk_idx [T, K] int32 (K = 0 allowed:
 * nothing is covered), driver [B] uint8, ctx_lens [B] int32, seq_lens [B]
 * int32.  Outputs: n_acc, event_row, new_cache_len int32 [B]; next_driver,
 * finished uint8 [B]; src uint8 [T].
 *
 * Errors: IPDV_EINVAL (null pointer, B < 0, K < 0 or K > IPDV_MAX_K), IPDV_EHIP.
 */
int accept_scan(const int32_t* cu_q, const int32_t* prop_tok,
                const int32_t* topk_idx, int K,
                const uint8_t* driver, const int32_t* ctx_lens, const int32_t* seq_lens,
                int32_t eos_id, int32_t max_len, int B,
                int32_t* n_acc, int32_t* event_row, uint8_t* next_driver,
                uint8_t* finished, int32_t* new_cache_len, uint8_t* src,
                void* hip_stream);

/*
 * accept_scan_rule -- accept_scan with the rule variants named after Eq. (9)
 * in Section 3.2.1 (SKD's behaviour as described in Section 2).
 *
 * take_rule (IPDV_TAKE_*) replaces the "uncovered" test of a student-driven
 * window and hand_rule (IPDV_HAND_*) the "covered" test of a teacher-driven
 * one; every other rule of accept_scan (first event ends the window, EOS,
 * length cap, cache lengths, source labels) is unchanged, with "covered"
 * read as "passes the takeover test" for a student EOS.
 *   IPDV_TAKE_ENTROPY: row i takes over when ent[row] > tau_take.
 *   IPDV_HAND_ENTROPY: row i hands back when ent[row] <= tau_hand.
 *     ent [T] float32 is a per-row entropy chosen by the caller (the paper
 *     allows the student's or the teacher's; e.g. the `entropy` output of
 *     lmhead_logsoftmax_verify for the verifier's).  Comparisons are IEEE: a
 *     NaN entropy passes neither test.
 *   IPDV_HAND_FIXED_ONE: a teacher-driven window keeps its first draft and
 *     hands back at row 0; a takeover's next driver stays S, since the
 *     replacement is the teacher's only token (SKD: the teacher resamples the
 *     rejected position and the student resumes).
 * With IPDV_TAKE_COVERAGE and IPDV_HAND_COVERAGE it equals accept_scan.
 *
 * ent may be NULL unless an entropy rule is selected; topk_idx may be NULL
 * when K = 0 or no coverage rule is selected.
 *
 * Errors: those of accept_scan, and IPDV_EINVAL for an unknown rule or a
 * NULL ent under an entropy rule.
 */
int accept_scan_rule(const int32_t* cu_q, const int32_t* prop_tok,
                     const int32_t* topk_idx, int K,
                     const uint8_t* driver, const int32_t* ctx_lens, const int32_t* seq_lens,
                     int32_t eos_id, int32_t max_len, int B,
                     int take_rule, int hand_rule, const float* ent,
                     float tau_take, float tau_hand,
                     int32_t* n_acc, int32_t* event_row, uint8_t* next_driver,
                     uint8_t* finished, int32_t* new_cache_len, uint8_t* src,
                     void* hip_stream);

/*
 * sample_takeover -- the teacher's replacement token at a takeover (Eq. (9),
 * second case: the uncovered student draft is discarded and the teacher
 * samples a replacement from its own distribution q(. | c_t) at that position;
 * Section 3.2.3: the rejected token is regenerated by the teacher).  The
 * verifier's logits at the takeover row are that distribution, so the draw
 * reuses the preceding lmhead_logsoftmax_verify call instead of a decode step.
 *
 * The call handles the sequences b = seq_ids[i], i < n_seq (seq_ids NULL: b =
 * i), and writes token / finished of those only, so that the calls of two
 * verifiers (two models, each with its own rows) compose.  For each such b
 * with driver[b] == IPDV_DRIVER_S and event_row[b] >= 0 (accept_scan's
 * outputs: a takeover at row j = event_row[b]) the row is r = cu_q[b] + j and
 * its hidden row m = row_local ? row_local[r] : r; then
 *   token[b] = the first vocabulary index v (index order) with
 *              sum_{w <= v} softmax(l_m)_w > u[b]      (temperature 1)
 * -- the inverse-CDF draw with the caller's uniform u[b] in [0, 1) -- and
 * finished[b] is set to 1 when token[b] == eos_id (a teacher EOS is accepted
 * directly).  The other handled sequences, and those whose m is negative or
 * not below M, get token -1 and keep their finished flag.
 *
 * hidden, W, M, Hd, V, K, dtype and workspace must be those of the preceding
 * lmhead_logsoftmax_verify call over the rows of hidden, with the workspace
 * unchanged since (its group records hold the mass of each 32-entry quarter
 * of each 128-entry group; the chosen quarter's 32 logits are recomputed
 * exactly).  seq_ids [n_seq] int32
 * or NULL; cu_q [B+1] int32, driver [B] uint8, event_row [B] int32, row_local
 * [T] int32 or NULL, u [B] float (B = the batch's sequences).  Outputs: token
 * int32 [B]; finished uint8 [B] (updated in place).
 * The draw agrees with the exact one whenever u[b] is farther than the fp32
 * rounding of the cumulative probabilities from an interval end (typically
 * about 1e-6 of the total mass; at most 1.2e-4 at V = 262144).
 *
 * Errors: IPDV_EINVAL (null pointer, n_seq < 0, the LM-head shape rules),
 * IPDV_EUNSUPPORTED, IPDV_EWORKSPACE, IPDV_EHIP.
 */
int sample_takeover(const void* hidden, const void* W, int M, int Hd, int V, int K,
                    const void* workspace, size_t workspace_bytes,
                    const int32_t* seq_ids, int n_seq,
                    const int32_t* cu_q, const uint8_t* driver, const int32_t* event_row,
                    const int32_t* row_local, const float* u, int32_t eos_id,
                    int32_t* token, uint8_t* finished, int dtype, void* hip_stream);

/*
 * lmhead_sample -- one draw per row from the model's distribution at
 * temperature 1, top-p 1 (Appendix A), reusing the preceding
 * lmhead_logsoftmax_verify call's group records: the proposer's sampling step
 * of the propose stage (Section 3.2.3: the driver proposes its next tokens
 * autoregressively; Eq. (9): x~ ~ pi(. | c_t) when the student drives, q when
 * the teacher does).
 *
 *   token[m] = the first vocabulary index v (index order) with
 *              sum_{w <= v} softmax(l_m)_w > u[m]
 * -- the inverse-CDF draw with the caller's uniform u[m] in [0, 1).
 *
 * hidden, W, M, Hd, V, K, dtype and workspace as in the preceding
 * lmhead_logsoftmax_verify call over these rows, the workspace unchanged
 * since.  u [M] float, token [M] int32.  The same rounding note as
 * sample_takeover applies.
 *
 * Errors: IPDV_EINVAL (null pointer, the LM-head shape rules),
 * IPDV_EUNSUPPORTED, IPDV_EWORKSPACE, IPDV_EHIP.
 */
int lmhead_sample(const void* hidden, const void* W, int M, int Hd, int V, int K,
                  const void* workspace, size_t workspace_bytes, const float* u,
                  int32_t* token, int dtype, void* hip_stream);

/*
 * lmhead_pack_w -- W [V, Hd] row-major bf16 -> the tiled layout of IPDV_W_TILED:
 * [ceil(V/16)][Hd/32][16][32], i.e. element (v, c) at
 * ((v/16) * (Hd/32) + c/32) * 512 + (v%16) * 32 + c%32, with rows V..16*ceil(V/16)-1
 * zero.  Each 16-row x 32-channel block is 1 KB contiguous, one pipeline
 * stage of the LM-head GEMM for 16 vocabulary rows.  Done once per weight
 * (at load time in an engine); the packed copy then replaces W in the calls
 * above with dtype IPDV_BF16 | IPDV_W_TILED.
 *
 * W_tiled: device buffer of ipdv_lmhead_packed_w_size(V, Hd) bytes, not
 * aliasing W.  V and Hd follow the LM-head shape rules.
 *
 * Errors: IPDV_EINVAL (null or aliasing pointers, shape rules),
 * IPDV_EUNSUPPORTED (dtype other than IPDV_BF16), IPDV_EHIP.
 */
size_t ipdv_lmhead_packed_w_size(int V, int Hd);
int lmhead_pack_w(const void* W, int V, int Hd, void* W_tiled, int dtype, void* hip_stream);

/*
 * lmhead_logp_gather -- log-softmax of a model's logits at listed vocabulary
 * indices: logp[m, j] = hidden[m] . W[idx[m, j]] - lse[m].  The union support
 * of Eq. (6) needs each model's log-probs at the other model's top-K indices
 * (S^pi u S^q, Eq. (5)); each model's own top-K log-probs come from
 * lmhead_logsoftmax_verify.
 *
 * hidden [M, Hd], W [V, Hd] (dtype), lse [M] float (that call's LSE for these
 * rows), idx [M, n_idx] int32, n_idx <= IPDV_MAX_GATHER.  Output logp [M,
 * n_idx] float; an index outside [0, V) gives -inf.  The dot product is
 * accumulated in fp32 in a different order from the GEMM's, so a value can
 * differ from the same index's top-K log-prob by fp32 rounding (about 1e-6
 * of the logit's magnitude).
 *
 * Errors: IPDV_EINVAL (null pointer, n_idx out of range, the LM-head shape
 * rules with K = 1), IPDV_EUNSUPPORTED, IPDV_EHIP.
 */
int lmhead_logp_gather(const void* hidden, const void* W, int M, int Hd, int V,
                       const float* lse, const int32_t* idx, int n_idx,
                       float* logp, int dtype, void* hip_stream);

/*
 * source_split_kl -- the per-position values of the source-split objective
 * (Section 3.2.2).  For each row m (a position c_t seen by both models):
 *   S^pi = s_idx[m, 0..K-1] (student top-K), S^q = t_idx[m, 0..K-1] (teacher);
 *   S_t  = the support (IPDV_SUPPORT_*; Eq. (5));
 *   pi_bar, q_bar = both distributions renormalised on S_t (Eq. (6));
 *   kl_rev[m] = D(pi_bar || q_bar), kl_fwd[m] = D(q_bar || pi_bar) (Eq. (10));
 *   loss[m]   = by src[m] and loss_mode (IPDV_LOSS_*): with the default,
 *               kl_rev where src = IPDV_SRC_S, kl_fwd where src = IPDV_SRC_T,
 *               0 where src = IPDV_SRC_DISCARDED;
 *   overlap[m] = |S^pi n S^q| / K (the top-K overlap ratio, Section 4.2).
 * An empty support (a disjoint intersection) gives 0 for both KLs.
 * With cu (segment offsets [B+1], one segment per trajectory), also
 *   seq_loss[b] = the mean of loss over the segment's emitted rows (src S or
 *                 T) -- the length-normalised inner term of Eq. (11);
 *   t_ratio[b]  = the share of teacher tokens among them (the intervention
 *                 ratio, Section 4.3); both 0 for a segment with none.
 *
 * Inputs, each [M, K] (float or int32): s_idx, s_logp (the student's top-K
 * and its log-probs, from its lmhead_logsoftmax_verify), s_at_t (the
 * student's log-probs at t_idx, from lmhead_logp_gather), t_idx, t_logp, t_at_s
 * (the same for the teacher); src [M] uint8.  Log-probs must be finite.  An
 * index in both lists takes its two log-probs from the list that defines the
 * support: the student's (s_logp, t_at_s) for the union, S^pi and the
 * intersection, the teacher's (s_at_t, t_logp) for S^q.  Outputs kl_rev,
 * kl_fwd, loss, overlap [M] and seq_loss, t_ratio [B] float are each
 * optional (NULL: not written); src is required with loss or cu, and loss
 * with cu and B > 0.  Computed in fp32.
 *
 * Errors: IPDV_EINVAL (null pointer, M < 0, K outside [1, IPDV_MAX_K], an
 * unknown support or loss mode, B < 0), IPDV_EHIP.
 */
int source_split_kl(int M, int K,
                    const int32_t* s_idx, const float* s_logp, const float* s_at_t,
                    const int32_t* t_idx, const float* t_logp, const float* t_at_s,
                    const uint8_t* src, int support, int loss_mode,
                    float* kl_rev, float* kl_fwd, float* loss, float* overlap,
                    const int32_t* cu, int B, float* seq_loss, float* t_ratio,
                    void* hip_stream);

/*
 * Optional timing hook for profilers and benchmarks (thread-local).  While
 * set, each kernel an entry point launches is bracketed by hipEventRecord of
 * the caller's events (hipEvent_t handles cast to void*), taken from
 * `events` in order: the first kernel of a call records one event before and
 * one after it, every further kernel one after it.  Recording stops when
 * `capacity` events are used.  NULL / 0 turns it off.  Returns IPDV_OK.
 * ipdv_trace_count() returns how many events have been recorded since the
 * hook was last set.  Intervals per call: verify_attn_paged 3 (append,
 * attention, split combine; on the bf16 D = 128 16-token-page path the
 * attention kernel appends the window itself and the append interval is
 * empty), lmhead_logsoftmax_verify 3 (the hidden rows' copy into the tiled
 * layout, empty where none is made; GEMM + epilogue; merge), accept_scan 1,
 * accept_scan_rule 1, sample_takeover 1, lmhead_sample 1, lmhead_pack_w 1,
 * lmhead_logp_gather 1, source_split_kl 1 (+1 with cu).
 */
int ipdv_trace_events(void* const* events, int capacity);
int ipdv_trace_count(void);

/* Thread-local description of the last non-OK status ("" if none). */
const char* ipdv_last_error(void);

/* Library version string. */
const char* ipdv_version(void);

#ifdef __cplusplus
}
#endif

#endif /* IPDV_H */
