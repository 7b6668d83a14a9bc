/*
 * dspark.h -- C ABI of the MI355X (gfx950) batched verification step of
 * confidence-scheduled speculative decoding (DSpark).
 *
 * Three stages, each a hand-written HIP kernel family:
 *   1. dspark_schedule    -- the hardware-aware prefix scheduler (Algorithm 1):
 *                            per-request verification lengths from draft
 *                            confidences and an engine throughput table;
 *   2. dspark_verify_attn -- ragged causal verify attention over a paged KV
 *                            cache (all verify tokens of all requests flattened
 *                            into one batch, as in the section on serving with
 *                            variable-length verification);
 *   3. dspark_accept      -- speculative acceptance (the speculative-decoding
 *                            background section): greedy match or stochastic
 *                            rejection sampling, emitting the accepted length
 *                            and the corrected / bonus token per request.
 * Upstream of them, the drafter's sequential stage (dspark_markov_draft,
 * dspark_rnn_draft) produces the draft tokens, distributions and confidences
 * they consume; dspark_check_*_inputs look at a call's device-side values
 * before it.
 *
 * Conventions shared by every entry point
 *   - All array arguments are DEVICE pointers unless marked "host".  Arrays are
 *     dense row-major unless strides are given.  The caller allocates and owns
 *     every buffer, including the workspace, sized with the matching
 *     *_workspace_size() call.  The library never allocates, frees or
 *     synchronises; it keeps no global state and is re-entrant.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream).
 *   - Arguments are validated on the host before anything touches the GPU;
 *     a failed check returns a non-zero dspark_status and enqueues nothing.
 *     dspark_last_error() then describes it (thread-local).  Values that live
 *     in device memory (lengths, tokens) cannot be checked on the host; the
 *     kernels clamp them into range as documented per call, so no access
 *     leaves the buffers described here -- except through block-table
 *     entries, which name pages of a cache whose size dspark_verify_attn is
 *     not told (dspark_check_verify_inputs checks them).
 *   - A workspace must not be shared by two calls that may run concurrently.
 */
#ifndef DSPARK_H
#define DSPARK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DSPARK_ABI_VERSION 3

typedef enum {
    DSPARK_OK = 0,
    DSPARK_EINVAL = 1,       /* null pointer / non-positive size / bad enum   */
    DSPARK_ESHAPE = 2,       /* sizes inconsistent with each other            */
    DSPARK_EDTYPE = 3,       /* unsupported element type                      */
    DSPARK_EUNSUPPORTED = 4, /* valid but outside what the kernels implement  */
    DSPARK_EWORKSPACE = 5,   /* workspace missing, too small or misaligned    */
    DSPARK_EHIP = 6          /* a HIP launch failed                           */
} dspark_status;

/* Element type codes.  The type is a plain 32-bit integer rather than an enum
   so that any value a caller passes is well defined to read (an unknown code
   is rejected with DSPARK_EDTYPE). */
typedef int32_t dspark_dtype;
enum { DSPARK_F32 = 0, DSPARK_BF16 = 1 };

/* A hipStream_t, passed opaquely. */
typedef void* dspark_stream;

/* Version of this ABI (DSPARK_ABI_VERSION of the built library). */
int dspark_abi_version(void);

/* Message for the last failed call on this thread ("" if none). */
const char* dspark_last_error(void);

/* ------------------------------------------------------------------------
 * Stage 1: hardware-aware prefix scheduler (Algorithm 1 of the section on
 * confidence-scheduled verification).
 *
 *   conf     [R, K] fp32   conditional confidence c_{r,j} of draft position
 *                          j+1 (confidence-head section).  The survival
 *                          probability a_{r,j} is the running product of
 *                          c_{r,1..j} in fp64, multiplied in increasing j.
 *                          A value that is not > 0 (0, negative, NaN) ends
 *                          request r's candidates; a value above 1 reads as 1.
 *   sps      [sps_len] fp64 engine throughput in steps/s at B verify tokens,
 *                          B = sum_r (1 + len_r); sps_len must be
 *                          > R*(K+1).  Entries below R are not read.
 *   mode     0 = the causal greedy with early stop (stop at the first
 *                admission that does not strictly raise Theta = tau * SPS(B));
 *            1 = no early stop: the best prefix of the same greedy path.
 *                On the CURRENT confidences this search is not lossless: the
 *                appendix counterexample shows it biasing the first output
 *                token, because later confidences depend on the realised
 *                drafts.  The lossless use of the no-break search is the
 *                asynchronous scheduler below (dspark_schedule_capacity on
 *                an earlier step's confidences, then dspark_schedule_topk).
 *   len      [R] int32 out  selected verification length l*_r in 0..K.
 *   cu_q     [R+1] int32 out (nullable) exclusive prefix sum of 1 + len_r:
 *                          request r's verify tokens are rows
 *                          cu_q[r] .. cu_q[r+1]-1 of the flattened batch.
 *   tok_req  [R*(K+1)] int32 out (nullable) request id of every flattened
 *                          verify token; slots >= cu_q[R] are set to -1.
 *   ws       workspace of dspark_schedule_workspace_size(R, K) bytes
 *                          (16 + 12*R*K, rounded up to 256), 256-aligned:
 *                          the candidates' admission positions and running
 *                          tau = R + sum of admitted a, passed from the
 *                          ranking kernel to the selection kernel.  Missing,
 *                          small or misaligned -> DSPARK_EWORKSPACE.
 *   The candidates (r, j) with a_{r,j} > 0 are admitted in descending a,
 *   ties by r then j.  Limits: 1 <= R, 0 <= K <= 64, R*K <= 8192.
 *   dspark_schedule_workspace_size returns 0 for sizes outside the limits.
 * ---------------------------------------------------------------------- */
size_t dspark_schedule_workspace_size(int R, int K);

dspark_status dspark_schedule(const float* conf, int R, int K, const double* sps,
                              int64_t sps_len, int mode, int32_t* len, int32_t* cu_q,
                              int32_t* tok_req, void* ws, size_t ws_bytes,
                              dspark_stream stream);

/* ------------------------------------------------------------------------
 * Stage 1 without a workspace argument, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  Arguments, outputs, limits and errors are those of
 * dspark_schedule.  The workspace is a fixed 98560-byte array in device memory
 * (the workspace of the largest schedule the limits allow, R*K = 8192), one
 * copy per GPU, held until the process ends; sizes needing more return
 * DSPARK_EWORKSPACE.  The call allocates nothing (no hipMalloc, hipFree or
 * allocating library routine); on its first call for a device it looks up the
 * array's address on that device (the device of `stream`).  Every call on one
 * GPU shares that GPU's array, so calls that may overlap on one GPU (two
 * streams, or two host threads) race and must not be issued; calls ordered on
 * one stream are safe.
 * ---------------------------------------------------------------------- */
dspark_status dspark_schedule_noalloc(const float* conf, int R, int K, const double* sps,
                                      int64_t sps_len, int mode, int32_t* len, int32_t* cu_q,
                                      int32_t* tok_req, dspark_stream stream);

/* ------------------------------------------------------------------------
 * Stage 1, asynchronous form (the section on the hardware-aware prefix
 * scheduler in practice).  The candidates of the current step are ranked by
 * their current survival products exactly as in dspark_schedule; only the
 * truncation length -- the capacity, a count of draft tokens -- comes from the
 * no-break search over the confidences of an earlier step (two steps before,
 * in the paper's pipeline).  Since the capacity cannot depend on the current
 * drafts, the admission of a draft does not depend on its own realisation.
 *
 * dspark_schedule_capacity: runs the no-break search (mode 1 above) on
 *   conf_prev [R, K] fp32 with the table sps [sps_len] fp64 (sps_len > R*(K+1))
 *   and writes the number of draft tokens it admits to *capacity (device
 *   int32).  It writes nothing else outside the workspace.
 * dspark_schedule_topk: admits the first min(*capacity, |E|) candidates of the
 *   current order (descending a of conf [R, K], ties by r then j; E = the
 *   candidates with a > 0; a negative capacity admits none) and writes len,
 *   cu_q and tok_req as dspark_schedule does.  *capacity is read on the device
 *   (typically written by an earlier dspark_schedule_capacity on the same
 *   stream), so the step needs no host round trip.  No throughput table is
 *   read.  With an unchanged request set the verify batch is R + *capacity
 *   tokens whenever |E| >= *capacity.
 * Both take the workspace of dspark_schedule_workspace_size(R, K) (256-aligned)
 * and the limits of dspark_schedule; null or misaligned pointers -> EINVAL.
 * ---------------------------------------------------------------------- */
dspark_status dspark_schedule_capacity(const float* conf_prev, int R, int K, const double* sps,
                                       int64_t sps_len, int32_t* capacity, void* ws,
                                       size_t ws_bytes, dspark_stream stream);

dspark_status dspark_schedule_topk(const float* conf, int R, int K, const int32_t* capacity,
                                   int32_t* len, int32_t* cu_q, int32_t* tok_req, void* ws,
                                   size_t ws_bytes, dspark_stream stream);

/* ------------------------------------------------------------------------
 * Stage 2: ragged causal verify attention over a paged KV cache (the target
 * model's verification forward pass over the flattened verify tokens).
 *
 *   q         [total_q, Hq, Dqk]  queries, total_q = cu_q[R].
 *   k_cache   paged keys:   element (page, head, slot, d) at
 *             page*k_strides[0] + head*k_strides[1] + slot*k_strides[2] + d.
 *   v_cache   paged values, likewise with v_strides; it may alias k_cache
 *             (latent attention: values are the first Dv <= Dqk dims).
 *   k_strides, v_strides  host int64[3], in elements.
 *   block_table [R, max_pages] int32: physical page of request r's logical
 *             page i (token j sits in page j / page_size, slot j % page_size).
 *   kv_len    [R] int32: context length of request r, INCLUDING its q_len_r
 *             verify tokens, which are its last q_len_r keys.  Query t of
 *             request r (0-based) attends keys 0 .. kv_len_r - q_len_r + t.
 *   cu_q      [R+1] int32: as produced by dspark_schedule.
 *   max_q     host bound on every q_len_r = cu_q[r+1] - cu_q[r] (K+1 after
 *             scheduling).  A request is skipped (its rows left unwritten)
 *             when q_len_r > max_q, when kv_len_r lies outside
 *             [q_len_r, max_pages*page_size], or when its rows cu_q[r] ..
 *             cu_q[r+1]-1 do not lie inside [0, min(cu_q[R], R*max_q)).
 *   Head h reads KV head h / (Hq / Hkv).
 *   scale     softmax scale, finite and > 0 (else DSPARK_EINVAL).
 *   out       [total_q, Hq, Dv] softmax(scale * q k^T) v in dtype `dt`
 *             (fp32 accumulation, rounded to nearest-even on store).
 *   lse       [total_q, Hq] fp32 (nullable): natural-log sum of exp of the
 *             scaled scores.
 *   dt        element type of q, k_cache, v_cache and out.
 *   Supported: Hq % Hkv == 0; Dqk, Dv multiples of 8 up to 576;
 *   page_size multiple of 16.  Which kernels run (results agree within the
 *   bf16 tolerance either way):
 *     - bf16, Dqk == Dv == 128, page_size a power of two >= 64, strides
 *       multiples of 8 elements, q/k/v 16-byte aligned: MFMA tiles, HBM-bound;
 *     - bf16, Dqk == 576, Dv == 512 (latent head), v_cache == k_cache with
 *       identical strides (values are the first 512 dims of the key rows),
 *       page_size a power of two >= 64, strides multiples of 8 elements,
 *       q/k/out 16-byte aligned: MFMA tiles, bound by the matrix cores;
 *     - anything else: vector ALUs.
 * ---------------------------------------------------------------------- */
size_t dspark_verify_attn_workspace_size(int R, int max_q, int Hq, int Hkv, int Dqk, int Dv,
                                         int max_pages, int page_size, dspark_dtype dt);

dspark_status dspark_verify_attn(const void* q, const void* k_cache, const void* v_cache,
                                 const int64_t* k_strides, const int64_t* v_strides,
                                 const int32_t* block_table, int max_pages,
                                 const int32_t* kv_len, const int32_t* cu_q, int R, int max_q,
                                 int Hq, int Hkv, int Dqk, int Dv, int page_size, float scale,
                                 dspark_dtype dt, void* out, float* lse, void* ws,
                                 size_t ws_bytes, dspark_stream stream);

/* ------------------------------------------------------------------------
 * Stage 3: speculative acceptance (the background section on speculative
 * decoding: left-to-right test, first rejection discards the suffix, one
 * corrected or bonus token per round).
 *
 *   draft_tok [R, K] int32: draft token for verify slot t+1 (the paper's
 *             x_{t+1}); values outside [0, V) are read as rejected.
 *   draft_p   [R, K, V] fp32 (nullable): draft distribution p_d for slot t+1,
 *             used as given (not renormalised); with K = 0 it may be NULL in
 *             stochastic mode too (u alone selects it).
 *   logits    target logits, row cu_q[r] + t (row stride `ld` elements) is the
 *             target distribution for the token after verify slot t:
 *             rows t < len_r test draft_tok[r, t]; row len_r gives the bonus.
 *   logit_dt  element type of logits.
 *   u         [R, K+1] fp32 uniforms in [0,1) (nullable): u[r,t] (t < K) tests
 *             draft t+1, u[r,K] draws the emitted token.
 *   cu_q      [R+1] int32 as produced by dspark_schedule; len_r = q_len_r - 1
 *             must lie in 0..K and the rows cu_q[r] .. cu_q[r+1]-1 inside
 *             [0, min(cu_q[R], R*(K+1))) (other requests get
 *             accepted_len = -1, next_tok = -1).
 *   draft_p == NULL and u == NULL: greedy -- draft t+1 is accepted iff it is
 *             the argmax of the raw logits of row t (lowest index on ties);
 *             the emitted token is the argmax of row accepted_len.
 *   otherwise stochastic -- p_t = softmax(inv_temperature * z); draft x is
 *             accepted iff u[r,t] < p_t(x) / p_d(x) (p_d(x) = 0 accepts); at
 *             the first rejection t* the emitted token is drawn from
 *             max(0, p_t - p_d) of row t* (p_t if that has no mass); with no
 *             rejection it is drawn from p_t of row len_r.  A draw is the
 *             smallest token v whose running mass (ascending v) exceeds
 *             u[r,K] times the total mass.
 *   accepted_len [R] int32 out, next_tok [R] int32 out.
 *   accept_rate  [total_q] fp32 out (nullable, stochastic only): for rows
 *             t < len_r the analytic acceptance probability
 *             sum_v min(p_t(v), p_d(v)) (one minus the total variation
 *             distance, the confidence head's training label); -1 for bonus
 *             rows and for rows that no request with len_r in 0..K owns.
 *   Limits: 1 <= V <= 2^20, ld >= V, 0 <= K <= 64, inv_temperature > 0.
 * ---------------------------------------------------------------------- */
size_t dspark_accept_workspace_size(int R, int K, int V);

dspark_status dspark_accept(const int32_t* draft_tok, const float* draft_p, const void* logits,
                            dspark_dtype logit_dt, int64_t ld, const float* u,
                            const int32_t* cu_q, int R, int K, int V, float inv_temperature,
                            int32_t* accepted_len, int32_t* next_tok, float* accept_rate,
                            void* ws, size_t ws_bytes, dspark_stream stream);

/* ------------------------------------------------------------------------
 * Drafter: the Markov-head draft block, which produces the inputs of the
 * three stages above (the sequential stage of semi-autoregressive drafting,
 * eq. sequential-factorization, with the Markov head of eq. markov, and the
 * confidence head of eq. confidence with the per-position temperatures of its
 * post-hoc calibration).  For every request r, with x_0 = anchor[r] and
 * k = 1 .. K, left to right:
 *     e_k = W1[x_{k-1}]                                  (rank-dim embedding)
 *     p_k = softmax(inv_temperature * (U_k + W2^T e_k))  (U_k: base logits)
 *     x_k = the smallest v whose running mass (ascending v) exceeds
 *           u[r, k-1] times the total mass
 *     c_k = sigmoid((w_h . h_k + w_e . e_k) / T_k)       (w_conf = [w_h; w_e])
 *
 *   anchor      [R] int32: x_0 (the last token of the previous verification).
 *   base_logits U_k of request r at element (r * K + k - 1) * ld; fp32 or
 *               bf16 (base_dt); ld >= V.
 *   W1          [V, rank] bf16 (uint16 bit patterns): embedding rows.
 *   W2t         [V, rank] bf16: the projection stored vocabulary-major, row v
 *               holding W2[:, v] (so a vocabulary tile is contiguous).
 *   rank        32, 64, 128 or 256 (the paper's default is 256).
 *   hidden      [R, K, d] bf16: the backbone state h_k of each position
 *               (nullable when d == 0).
 *   w_conf      [d + rank] fp32: confidence weights, hidden part first.
 *   sts_temp    [K] fp32 per-position temperatures T_k (nullable: all 1).
 *   u           [R, K] fp32 uniforms in [0, 1), one per draw.
 *   draft_tok   [R, K] int32 out: x_1 .. x_K (dspark_accept's draft_tok).
 *   draft_p     [R, K, V] fp32 out: p_1 .. p_K (dspark_accept's draft_p).
 *   conf        [R, K] fp32 out: c_1 .. c_K (dspark_schedule's conf).
 *   An anchor outside [0, V) marks its request invalid: its draft_tok row is
 *   -1 and its conf row NaN (its draft_p rows hold finite values computed
 *   with embedding row 0).
 *   Limits: 1 <= R <= 8192, 1 <= K <= 64, 1 <= V <= 262144, 0 <= d <= 2^16,
 *   inv_temperature > 0; W1, W2t 16-byte aligned.  The base logits and
 *   draft_p are read and written four entries at a time when V and ld are
 *   multiples of 4 and the rows are aligned, else one at a time.
 * ---------------------------------------------------------------------- */
size_t dspark_markov_draft_workspace_size(int R, int K, int V, int rank);

dspark_status dspark_markov_draft(const int32_t* anchor, const void* base_logits,
                                  dspark_dtype base_dt, int64_t ld, const uint16_t* W1,
                                  const uint16_t* W2t, int rank, const uint16_t* hidden,
                                  const float* w_conf, int d, const float* sts_temp,
                                  const float* u, float inv_temperature, int R, int K, int V,
                                  int32_t* draft_tok, float* draft_p, float* conf, void* ws,
                                  size_t ws_bytes, dspark_stream stream);

/* ------------------------------------------------------------------------
 * Drafter, RNN head: the same draft block with the RNN head of the section on
 * semi-autoregressive generation (eq. rnn) in place of the Markov head.  A
 * recurrent state carries the whole prefix of the block.  For every request
 * r, with x_0 = anchor[r], s_0 = 0 and k = 1 .. K, left to right:
 *     e_k = W1[x_{k-1}],   z_k = [s_{k-1}; e_k; h_k]        (2 rank + d values)
 *     a_k = Wrnn z_k = [a_g; a_c; a_o]                      (3 rank values)
 *     s_k = sigmoid(a_g) * s_{k-1} + (1 - sigmoid(a_g)) * tanh(a_c)
 *     p_k = softmax(inv_temperature * (U_k + W2^T tanh(a_o)))
 *     x_k, c_k as for dspark_markov_draft (c_k reads [h_k; e_k]).
 *
 *   Wrnn  [3 rank, 2 rank + d] bf16 row-major, 16-byte aligned: the single
 *         projection of the equation, rows 0 .. rank-1 the gate, then the
 *         candidate, then the output component; columns in the order of z_k.
 *         The equation has no bias terms.
 *   Every other argument, output, limit and the invalid-anchor rule are those
 *   of dspark_markov_draft, and in addition d % 8 == 0 and hidden 16-byte
 *   aligned when d > 0 (the backbone part of the projection, Wrnn[:, 2 rank:]
 *   h_k, runs on the matrix cores once for every position).  The state and
 *   the head's output are fp32; the output enters the bf16 vocabulary product
 *   as three bf16 terms whose sum is its fp32 value.
 *   ws    dspark_rnn_draft_workspace_size(R, K, V, rank) bytes, 256-aligned.
 * ---------------------------------------------------------------------- */
size_t dspark_rnn_draft_workspace_size(int R, int K, int V, int rank);

dspark_status dspark_rnn_draft(const int32_t* anchor, const void* base_logits,
                               dspark_dtype base_dt, int64_t ld, const uint16_t* W1,
                               const uint16_t* W2t, const uint16_t* Wrnn, int rank,
                               const uint16_t* hidden, const float* w_conf, int d,
                               const float* sts_temp, const float* u, float inv_temperature,
                               int R, int K, int V, int32_t* draft_tok, float* draft_p,
                               float* conf, void* ws, size_t ws_bytes, dspark_stream stream);

/* ------------------------------------------------------------------------
 * Input checks: the device-side values of a call, looked at before it.
 *
 * The stages clamp the values that live in device memory so that no access
 * leaves the buffers described above, and skip the requests that break a
 * rule; two kinds of value cannot be caught that way.  A block-table entry
 * names a page of a cache whose size dspark_verify_attn is not told, so an
 * entry past the cache is read as if it were a page; and a uniform or a
 * confidence outside its range changes the result without any access going
 * astray.  Each check enqueues one small kernel on `stream` (nothing is
 * synchronised) that writes the first rule broken -- the smallest request
 * index, then the rule order below -- to `report`, a device int32[4]:
 *   {code, request, index, value}, code 0 = every rule holds.
 * The caller reads it once the stream has run the check, before the call it
 * guards.  Bad sizes or pointers -> EINVAL with nothing enqueued.
 *
 * dspark_check_verify_inputs (dspark_verify_attn's block_table, max_pages,
 * kv_len, cu_q, R, max_q, page_size, and num_pages, the number of pages of
 * the cache): code 1 rows cu_q[r] .. cu_q[r+1]-1 not inside
 * [0, min(cu_q[R], R*max_q)) or cu_q decreasing (index 0: value cu_q[r];
 * 1: cu_q[r+1]); 2 q_len_r above max_q (value q_len_r); 3 kv_len_r outside
 * [q_len_r, max_pages*page_size] (value kv_len_r); 4 a block-table entry of a
 * page the request reads outside [0, num_pages) (index: logical page, value:
 * the entry).
 * dspark_check_accept_inputs (dspark_accept's cu_q, u (nullable), R, K):
 * code 1 rows as above with R*(K+1); 2 len_r = q_len_r - 1 outside [0, K];
 * 3 u[r, t] (t = 0 .. K) outside [0, 1) or NaN (index t, value: the float's
 * bits).
 * dspark_check_schedule_inputs (dspark_schedule's conf, R, K): code 1
 * conf[r, j] outside [0, 1] or NaN (index j, value: the float's bits).
 * dspark_check_draft_inputs (dspark_markov_draft's and dspark_rnn_draft's u,
 * sts_temp (nullable), R, K): code 1 a temperature sts_temp[k] not finite and
 * positive (request -1, index k, value: the float's bits); 2 u[r, k] outside
 * [0, 1) or NaN (index k, value: the float's bits).
 * ---------------------------------------------------------------------- */
dspark_status dspark_check_verify_inputs(const int32_t* block_table, int max_pages,
                                         const int32_t* kv_len, const int32_t* cu_q, int R,
                                         int max_q, int page_size, int num_pages, int32_t* report,
                                         dspark_stream stream);

dspark_status dspark_check_accept_inputs(const int32_t* cu_q, const float* u, int R, int K,
                                         int32_t* report, dspark_stream stream);

dspark_status dspark_check_schedule_inputs(const float* conf, int R, int K, int32_t* report,
                                           dspark_stream stream);

dspark_status dspark_check_draft_inputs(const float* u, const float* sts_temp, int R, int K,
                                        int32_t* report, dspark_stream stream);

#ifdef __cplusplus
}
#endif
#endif /* DSPARK_H */
