/*
 * mdss.h -- C ABI of the MI355X (gfx950) multi-draft selection library.
 *
 * Method: Khisti et al., "Multi-Draft Speculative Sampling: Canonical
 * Decomposition and Theoretical Limits" (ICLR 2025).  Theorem 1 splits the
 * token-level selection of one output token from K drafted tokens into
 *   (1) importance weighted sampling (Definition 1) of one intermediate token
 *       Y among the drafts, here with the classical weights named right after
 *       Definition 1: Pr(I = i | x_1..x_K) proportional to w(x_i), and
 *   (2) single-draft speculative sampling (Algorithm 1, appendix on
 *       speculative decoding) of Y against the target, with the induced
 *       distribution r of Y in the role of the draft distribution.
 *
 * Notation used throughout this library: p = TARGET distribution, q = DRAFT
 * distribution, w(x) = p(x)/q(x).  (The paper uses the letters the other way
 * round: its p is the draft model and its q the target model.)
 *
 * Conventions shared by every entry point:
 *   - p, q, r and residual are row-major [B][V] fp32 arrays in device memory,
 *     rows contiguous (leading dimension V).  They are read as given: rows
 *     are not renormalised.
 *   - All pointers are HIP device pointers unless stated otherwise.  The
 *     caller owns every buffer, including the workspace; the library never
 *     allocates, frees or keeps device memory between calls (the one
 *     exception: the fixed scratch array of mdss_induced_dist_expsum_noalloc).
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     Every call only enqueues work on it and returns; the caller
 *     synchronises.  Calls on one stream run in issue order.
 *   - Argument errors (null pointer, bad size, K or workspace) are returned
 *     synchronously before anything is launched, and nothing is written.
 *     A failed launch returns MDSS_EDEVICE.
 *   - B = 0 is an empty batch: once the sizes and the other parameters
 *     (K, s_max, s, tail, m) have been checked, the call returns MDSS_OK
 *     without reading, writing or launching anything; its pointers and its
 *     workspace may then be NULL, and the workspace-size queries return 0.
 *   - Per-row data problems are reported in row_status[b] (nullable), as bits
 *     OR-ed into the existing value: the caller zeroes row_status before the
 *     first call of a step.  A flagged row gets r = NaN and token -1.
 *   - Uniforms: u is [B][3] fp32 (device): u[b][0] for the selection draw,
 *     u[b][1] for the accept test, u[b][2] for the residual draw, each in
 *     [0, 1).  If u is NULL they are generated on the device from
 *     Philox4x32-10 (Salmon et al., SC'11) with key = seed and counter =
 *     (offset + b) (low word first, upper two counter words zero): output
 *     word j gives u_j = (word_j >> 8) * 2^-24.
 */
#ifndef MDSS_H
#define MDSS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum mdss_status {
  MDSS_OK = 0,
  MDSS_EINVAL = 1,       /* null pointer or invalid argument value */
  MDSS_ESHAPE = 2,       /* B outside [0, MDSS_MAX_B] or V outside [2, MDSS_MAX_V] */
  MDSS_EUNSUPPORTED = 3, /* K outside {2, 3} for mdss_induced_dist, outside [2, MDSS_MAX_K] for
                            the selection and the exponential-sum calls (MDSS_SUCCESSIVE_MAX_K for
                            the successive calls), K = 3 with s_max outside [1, MDSS_K3_MAX_SUPPORT],
                            or a truncated-LP s outside [1, MDSS_TLP_MAX_S] */
  MDSS_EDEVICE = 4,      /* a HIP call or kernel launch failed */
  MDSS_EWORKSPACE = 5    /* workspace missing or smaller than mdss_workspace_bytes(), or (allocation-free
                            call) sizes beyond MDSS_NOALLOC_SCRATCH_BYTES */
} mdss_status;

/* row_status bits */
#define MDSS_ROW_BAD_PROB 1  /* NaN, infinite or negative probability in the row (or in p/q at a draft) */
#define MDSS_ROW_BAD_DRAFT 2 /* drafted / selected token out of [0, V) or with q = 0 */
#define MDSS_ROW_SUPPORT 4   /* K = 3: more than s_max tokens with q > 0 */
#define MDSS_ROW_FORCED 8    /* rejection with zero residual mass: the selected token is output */
#define MDSS_ROW_LP_LIMIT 16 /* truncated LP stopped after its augmentation limit (result feasible, maybe not optimal) */
#define MDSS_ROW_RANGE 32    /* exponential-sum calls: the row's positive weights span more than 2^300 (possible
                                only with probabilities far above 1); r = NaN */

#define MDSS_MAX_V 8388608LL /* rows longer than 2^23 tokens are rejected with MDSS_ESHAPE */
#define MDSS_MAX_B 65535LL   /* at most 65535 positions per call */
#define MDSS_K3_MAX_SUPPORT 4096 /* largest s_max accepted for K = 3 */
#define MDSS_MAX_K 8         /* largest K of the direct K-draft selection and of mdss_induced_dist_expsum */

/* Bytes of device workspace mdss_induced_dist needs for these sizes
 * (0 if the arguments are invalid or B = 0).  The workspace is caller-owned scratch:
 * its content on entry is ignored and on exit is unspecified. */
size_t mdss_workspace_bytes(int64_t B, int64_t V, int32_t K, int32_t s_max);

/* Induced distribution r of the selected token (step 1 of Theorem 1), for K
 * i.i.d. drafts from q and the classical importance weights w = p/q:
 *   r(y) = sum over ordered draft tuples x of prod_i q(x_i) * beta_y(x),
 *   beta_y(x) = sum over i with x_i = y of w(x_i) / sum_j w(x_j)
 * (Definition 1; the marginal in the proof of Theorem 1).  For K = 2 this is
 * the pair form of the selected-token distribution (eq. p_Ieq0) with
 * w_{k,i} = w(k)/(w(k)+w(i)).  The library evaluates it through the
 * exchangeable form
 *   r(y) = K p(y) sum_{x_2..x_K in supp q} prod_j q(x_j) / (w(y) + sum_j w(x_j))
 * for q(y) > 0, p(y) > 0; r(y) = q(y) Q0^(K-1) for q(y) > 0, p(y) = 0 (Q0 =
 * draft mass of such zero-weight tokens: all weights of such a tuple are zero
 * and the index is then chosen uniformly); r(y) = 0 for q(y) = 0.
 *   K = 2: O(n^2) pair sum per row, n = |supp q| <= V.
 *   K = 3: O(n^3) triple sum, only for rows with n <= s_max (else the row is
 *          flagged MDSS_ROW_SUPPORT): use it on top-s truncated draft rows.
 * p, q: [B][V] in; r: [B][V] out (every entry written).  s_max is ignored for
 * K = 2.  workspace: device buffer of at least mdss_workspace_bytes(B, V, K,
 * s_max) bytes, 256-byte aligned. */
mdss_status mdss_induced_dist(const float* p, const float* q, int64_t B, int64_t V, int32_t K, int32_t s_max,
                              float* r, int32_t* row_status, void* workspace, size_t workspace_bytes, void* stream);

/* Importance weighted selection of one drafted index (Definition 1, index form
 * with the classical weights).  For row b with drafts x_1..x_K (drafts is
 * [B][K] int32), w_i = p(x_i)/q(x_i) in fp64, W = w_1 + ... + w_K, running
 * sums C_i = w_1 + ... + w_i (left to right); the selected index is the
 * smallest i with u_sel * W < C_i, or floor(u_sel * K) when W = 0.
 * sel_index and sel_token ([B] int32 out) receive i (0-based) and x_i, or -1
 * for a row whose drafts are invalid (MDSS_ROW_BAD_DRAFT / MDSS_ROW_BAD_PROB).
 * u may be NULL (Philox, see above).  K in [2, MDSS_MAX_K]. */
mdss_status mdss_select_intermediate(const float* p, const float* q, const int32_t* drafts, const float* u,
                                     uint64_t seed, uint64_t offset, int64_t B, int64_t V, int32_t K,
                                     int32_t* sel_index, int32_t* sel_token, int32_t* row_status, void* stream);

/* Single-draft speculative sampling of the selected token Y = sel_token[b]
 * against the target, with r as the proposal distribution (Algorithm 1):
 *   accept iff u_acc * r(Y) < p(Y)   (fp64; exact for fp32 r, p and a 24-bit u),
 *   otherwise output the smallest token j with C_j > u_res * Z, where
 *   res(x) = max(0, p(x) - r(x)) in fp64, Z = sum_x res(x) and C_j the running
 *   sum in ascending token id.  Z = 0 on a rejection: output Y, accepted = 1,
 *   MDSS_ROW_FORCED.
 * out_token [B] int32 and accepted [B] uint8 are outputs (-1 / 0 for an
 * invalid row: Y = -1, Y out of range, or NaN/negative/inf in p or r).
 * residual ([B][V] fp32, nullable) receives res for every row and
 * residual_mass ([B] fp64, nullable) receives Z; when both are NULL, rows
 * whose token is accepted do not read p or r beyond p(Y), r(Y).
 * workspace: device buffer of at least mdss_workspace_bytes_accept(B, V)
 * bytes, 256-byte aligned (room for one fp64 residual sum per 256 tokens, or
 * four per 1024 tokens, of every position): when a residual output is asked for, a row's residual is
 * summed by one workgroup per 4096-token segment and the draw reads the sums
 * of its row (two launches); otherwise one workgroup per position reads its
 * drafts' entries and, if it rejects, its own row (one launch). */
size_t mdss_workspace_bytes_accept(int64_t B, int64_t V);

mdss_status mdss_accept_or_resample(const float* p, const float* r, const int32_t* sel_token, const float* u,
                                    uint64_t seed, uint64_t offset, int64_t B, int64_t V, int32_t* out_token,
                                    uint8_t* accepted, float* residual, double* residual_mass, int32_t* row_status,
                                    void* workspace, size_t workspace_bytes, void* stream);

/* Selection and single-draft speculative sampling in one call (Theorem 1:
 * select the intermediate token, then run Algorithm 1 against r).  Outputs,
 * row flags and every written value are those of mdss_select_intermediate
 * followed by mdss_accept_or_resample with the same p, q, drafts, u, seed and
 * offset (the selected token is passed on inside the launch); sel_index and
 * sel_token ([B] int32) are nullable here.  r is the proposal of the selected
 * token ([B][V] fp32, e.g. from mdss_induced_dist_expsum).  K in
 * [2, MDSS_MAX_K].  The draft values p(x_i), q(x_i), r(x_i) are read
 * together, so the accept test waits for one round of loads after the
 * drafts.  workspace as for mdss_accept_or_resample. */
mdss_status mdss_select_accept(const float* p, const float* q, const float* r, const int32_t* drafts,
                               const float* u, uint64_t seed, uint64_t offset, int64_t B, int64_t V, int32_t K,
                               int32_t* sel_index, int32_t* sel_token, int32_t* out_token, uint8_t* accepted,
                               float* residual, double* residual_mass, int32_t* row_status, void* workspace,
                               size_t workspace_bytes, void* stream);

/* Theorem 1's two steps sharing one pass over the rows.
 * mdss_induced_dist_expsum_sums: r as mdss_induced_dist_expsum (the same
 * kernels, bit-identical r and row flags), and, from the same pass, the sums
 * Algorithm 1 with proposal r needs: for every position and 1024-token
 * sub-tile, four fp64 partial sums of res(x) = max(0, p(x) - r(x)) (NaN where
 * a p or r is not a probability), written into accept_workspace (at least
 * mdss_workspace_bytes_accept(B, V) bytes).  Unlike every other call, it SETS
 * row_status[b] (nullable) to its own flags instead of OR-ing them in, so the
 * status words need no clearing before it (it is the first call of a step).
 * mdss_select_accept_sums: selection and Algorithm 1 as mdss_select_accept,
 * with Z and the running sums taken from those partial sums instead of a pass
 * over the rows (the crossing sub-tile's 1024 entries are read again to find
 * the token); residual_mass (nullable) receives Z; there is no residual
 * output.  accept_workspace must hold the sums of the last
 * mdss_induced_dist_expsum_sums (or mdss_induced_dist_topk_expsum_sums) call,
 * with p and r unchanged since.  The
 * selection, the accept decision, the flags and Z agree with
 * mdss_select_accept; Z and the running sums are the same fp64 sums taken in
 * another order, so a resampled token can differ only where u_res Z lies
 * within the rounding of an fp64 sum of a CDF edge. */
mdss_status mdss_induced_dist_expsum_sums(const float* p, const float* q, int64_t B, int64_t V, int32_t K, float* r,
                                          int32_t* row_status, void* workspace, size_t workspace_bytes,
                                          void* accept_workspace, size_t accept_workspace_bytes, void* stream);
mdss_status mdss_select_accept_sums(const float* p, const float* q, const float* r, const int32_t* drafts,
                                    const float* u, uint64_t seed, uint64_t offset, int64_t B, int64_t V, int32_t K,
                                    int32_t* sel_index, int32_t* sel_token, int32_t* out_token, uint8_t* accepted,
                                    double* residual_mass, int32_t* row_status, void* accept_workspace,
                                    size_t accept_workspace_bytes, void* stream);

/* ---- Two drafts from different distributions (K = 2) --------------------
 * Remark 1 (and the non-identical K = 2 appendix): X1 ~ q1 and X2 ~ q2
 * independently.  The classical weight of draft i is w_i(x) = p(x)/q_i(x),
 * the target over the distribution that proposed it, and
 * Pr(I = i | x1, x2) = w_i(x_i) / (w_1(x1) + w_2(x2)) (uniform when both are
 * zero).  The induced distribution is
 *   r(y) = p(y) [ sum_{x in supp q2} q2(x) / (w_1(y) + w_2(x))      (if q1(y) > 0)
 *               + sum_{x in supp q1} q1(x) / (w_1(x) + w_2(y)) ]    (if q2(y) > 0)
 * and, for p(y) = 0, r(y) = (q1(y) Q2_0 + q2(y) Q1_0) / 2, Qi_0 = q_i-mass of
 * the tokens with p = 0.  Two O(n1 n2) sums per row.  Same conventions and
 * errors as the identical-draft calls; q1, q2 are [B][V] fp32. */
size_t mdss_workspace_bytes_pair(int64_t B, int64_t V);

mdss_status mdss_induced_dist_pair(const float* p, const float* q1, const float* q2, int64_t B, int64_t V, float* r,
                                   int32_t* row_status, void* workspace, size_t workspace_bytes, void* stream);

/* Selection between drafts[b][0] ~ q1 and drafts[b][1] ~ q2: w_1 = p(x1)/q1(x1),
 * w_2 = p(x2)/q2(x2) in fp64; index 0 iff u_sel (w_1 + w_2) < w_1; both zero:
 * floor(2 u_sel).  Outputs and row flags as mdss_select_intermediate. */
mdss_status mdss_select_intermediate_pair(const float* p, const float* q1, const float* q2, const int32_t* drafts,
                                          const float* u, uint64_t seed, uint64_t offset, int64_t B, int64_t V,
                                          int32_t* sel_index, int32_t* sel_token, int32_t* row_status,
                                          void* stream);

/* mdss_select_intermediate_pair followed by mdss_accept_or_resample in one
 * call, as mdss_select_accept is for identical drafts (drafts [B][2]). */
mdss_status mdss_select_accept_pair(const float* p, const float* q1, const float* q2, const float* r,
                                    const int32_t* drafts, const float* u, uint64_t seed, uint64_t offset,
                                    int64_t B, int64_t V, int32_t* sel_index, int32_t* sel_token,
                                    int32_t* out_token, uint8_t* accepted, float* residual, double* residual_mass,
                                    int32_t* row_status, void* workspace, size_t workspace_bytes, void* stream);

/* ---- Successive pairwise selection (K >= 2) -------------------------------
 * Remark 4: K drafts X1..XK i.i.d. from q are reduced two at a time.  Stage 1
 * selects between X1 and X2 as mdss_select_intermediate does for K = 2 and
 * keeps Y1, whose law is r_1 = the K = 2 induced distribution; stage j >= 2
 * selects between Y_{j-1} (law r_{j-1}) and X_{j+1} (law q) as two drafts of
 * different distributions (mdss_induced_dist_pair with q1 = r_{j-1}, q2 = q),
 * and keeps Y_j with law r_j.  r_{K-1} is the proposal of Algorithm 1.  Each
 * stage's law is used in its fp32 storage by the next stage.  Cost: K - 1
 * pair sums of O(n^2) per row, against O(n^K) for the direct K-draft rule. */
#define MDSS_SUCCESSIVE_MAX_K 8

/* Workspace bytes of mdss_induced_dist_successive (0 if the shape is invalid or B = 0). */
size_t mdss_workspace_bytes_successive(int64_t B, int64_t V);

/* r_stages: [K-1][B][V] fp32 out, stage j (1-based) at offset (j-1) B V; the
 * last stage is the proposal.  K in [2, MDSS_SUCCESSIVE_MAX_K].  Row flags as
 * mdss_induced_dist (a flagged row is NaN in every later stage).  workspace: at
 * least mdss_workspace_bytes_successive(B, V) bytes, 256-byte aligned. */
mdss_status mdss_induced_dist_successive(const float* p, const float* q, int64_t B, int64_t V, int32_t K,
                                         float* r_stages, int32_t* row_status, void* workspace,
                                         size_t workspace_bytes, void* stream);

/* Chained selection over drafts [B][K]: stage 1 keeps X1 iff u_1 (w1 + w2) < w1
 * with w_i = p(X_i)/q(X_i); stage j >= 2 keeps Y iff u_j (wY + wX) < wY with
 * wY = p(Y)/r_{j-1}(Y), wX = p(X_{j+1})/q(X_{j+1}); both weights zero: keep iff
 * floor(2 u_j) = 0 (fp64 throughout).  u_sel: [B][K-1] fp32 (u_j = u_sel[b][j-1])
 * or NULL: u_j from word 0 of Philox4x32-10 with key = seed and counter =
 * (offset + b (low, high word), j, 0), a stream apart from the one the other
 * calls use (third counter word 0).  sel_index = the draft index finally kept,
 * sel_token its id; -1 for a row with an invalid draft (out of range, q = 0, or
 * a kept token whose stage law is 0 or NaN: MDSS_ROW_BAD_DRAFT) or a NaN /
 * negative p or q at a draft (MDSS_ROW_BAD_PROB).  r_stages may be NULL for K = 2. */
mdss_status mdss_select_successive(const float* p, const float* q, const float* r_stages, const int32_t* drafts,
                                   const float* u_sel, uint64_t seed, uint64_t offset, int64_t B, int64_t V,
                                   int32_t K, int32_t* sel_index, int32_t* sel_token, int32_t* row_status,
                                   void* stream);

/* ---- Induced distribution by an exponential-sum quadrature ---------------
 * The same r as mdss_induced_dist (K i.i.d. drafts), mdss_induced_dist_pair
 * (two draft laws) and mdss_induced_dist_successive (successive pairwise),
 * evaluated in O(n) per node instead of O(n^K) per row.  Every denominator D
 * of those sums (a sum of positive weights) enters through
 *   1/D = integral over t of exp(t - D e^t) dt,
 * so for K i.i.d. drafts
 *   r(y) = K p(y) integral of e^t exp(-e^t w(y)) S(e^t)^(K-1) dt,
 *   S(a) = sum_{x in supp q} q(x) exp(-a w(x)),
 * and the two-law sums factor the same way.  The integral is taken by the
 * trapezoidal rule with step 1/2 on t, cut where both tails are below 1e-8
 * of every denominator of the row: about (ln(D_max/D_min) + 21.3) * 2 nodes
 * (60 on LLM-like rows).  Per token, nodes with a w <= 1/4 enter through an
 * eight-term expansion and nodes with a w > 22 are dropped; a token's nine node
 * terms and its expansion are evaluated together as one degree-10 polynomial in
 * its a_k0 w (k0 its first node with a w > 1/4, so a_k0 w lies in (1/4, e^(1/2)/4]).
 * Relative error of every entry, all terms being positive: at most
 * 2 sum_m |Gamma(1 + 4 pi i m)| = 4.8e-8 for the rule, 2e-8 for the grid's
 * tails, 7e-9 for the dropped nodes, 1e-9 for the expansion and 4.7e-9 for the
 * polynomial, 8.1e-8 in all, plus fp32 rounding (a row with a
 * ratio outside the fp32 normal range, or whose weights span more than 2^160
 * within 4096 tokens, is evaluated in fp64).  The zero-weight closed forms are
 * the ones stated above.  Any K in
 * [2, MDSS_MAX_K] (no support cap).  A row whose weights span more than 2^300
 * is flagged MDSS_ROW_RANGE (r = NaN); other flags and outputs as
 * mdss_induced_dist.  Workspace: caller-owned, 256-byte aligned. */

/* Bytes of workspace for mdss_induced_dist_expsum (0 if the arguments are invalid or B = 0). */
size_t mdss_workspace_bytes_expsum(int64_t B, int64_t V, int32_t K);

/* r: [B][V] fp32 out, the induced distribution of K i.i.d. drafts from q with
 * the classical weights (as mdss_induced_dist, for any K in [2, MDSS_MAX_K]). */
mdss_status mdss_induced_dist_expsum(const float* p, const float* q, int64_t B, int64_t V, int32_t K, float* r,
                                     int32_t* row_status, void* workspace, size_t workspace_bytes, void* stream);

/* ---- Allocation-free variant (for callers that cannot allocate) ----------
 * For callers that cannot call hipMalloc or take a caller-owned workspace:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * device allocation.  The same computation as mdss_induced_dist_expsum (same
 * kernels, bit-identical outputs and row flags), with its workspace in a fixed
 * device array of MDSS_NOALLOC_SCRATCH_BYTES inside the library: every GPU the
 * library runs on holds one copy of it from the first call made on that GPU
 * until the process ends.  The call allocates and frees nothing.
 *   - Sizes whose workspace (mdss_workspace_bytes_expsum(B, V, K)) exceeds
 *     MDSS_NOALLOC_SCRATCH_BYTES are rejected with MDSS_EWORKSPACE before
 *     anything is launched (256 positions of 32000 tokens need 26.2 MiB).
 *   - Every call on one GPU uses that GPU's one array: calls that overlap on a
 *     GPU (several streams, several host threads) race on it and must be
 *     ordered by the caller.  The array keeps the last call's contents; no call
 *     depends on them.
 *   - The first call on a device looks the array's device address up
 *     (hipGetSymbolAddress) with that device current; a failure there returns
 *     MDSS_EDEVICE.
 * Arguments, errors and outputs otherwise as mdss_induced_dist_expsum. */
#define MDSS_NOALLOC_SCRATCH_BYTES (32LL << 20)

mdss_status mdss_induced_dist_expsum_noalloc(const float* p, const float* q, int64_t B, int64_t V, int32_t K,
                                             float* r, int32_t* row_status, void* stream);

/* r: [B][V] fp32 out, the induced distribution of K i.i.d. drafts from a draft
 * truncated to at most s_max tokens (the top-s setting of mdss_induced_dist for
 * K = 3): the r of mdss_induced_dist_expsum, by the same trapezoidal rule on
 * the same node grid, with every (node, token) term of S(a_k) and of each
 * token's sum taken directly over the support (no windows, expansions or
 * polynomial tables), so its error is the rule's 4.8e-8 and the grid's 2e-8
 * plus rounding.  One workgroup per row streams p and q once and holds the
 * row's support on chip.
 *   - A row with more than s_max tokens of q > 0 is flagged MDSS_ROW_SUPPORT
 *     and gets r = NaN, as mdss_induced_dist does for K = 3; other flags
 *     (MDSS_ROW_BAD_PROB, MDSS_ROW_RANGE) and outputs as
 *     mdss_induced_dist_expsum.
 *   - K in [2, MDSS_MAX_K], s_max in [1, MDSS_K3_MAX_SUPPORT] (else
 *     MDSS_EUNSUPPORTED).  No workspace: the call allocates nothing. */
mdss_status mdss_induced_dist_topk_expsum(const float* p, const float* q, int64_t B, int64_t V, int32_t K,
                                          int32_t s_max, float* r, int32_t* row_status, void* stream);

/* The summed form of the top-s call (Theorem 1's two steps sharing one pass,
 * as mdss_induced_dist_expsum_sums): r bit-identical to
 * mdss_induced_dist_topk_expsum, and, from the same pass over the row, the
 * residual sums Algorithm 1 with proposal r needs, in the layout
 * mdss_select_accept_sums reads (four fp64 partial sums of max(0, p - r) per
 * 1024-token sub-tile, NaN for a flagged row), written into accept_workspace
 * (at least mdss_workspace_bytes_accept(B, V) bytes).  It SETS row_status[b]
 * (nullable) to its own flags.
 * Then call mdss_select_accept_sums with the same p, q, r and workspace. */
mdss_status mdss_induced_dist_topk_expsum_sums(const float* p, const float* q, int64_t B, int64_t V, int32_t K,
                                               int32_t s_max, float* r, int32_t* row_status, void* accept_workspace,
                                               size_t accept_workspace_bytes, void* stream);

/* The whole step of the top-s call in one launch (Theorem 1's selection, then
 * Algorithm 1 with proposal r): mdss_induced_dist_topk_expsum_sums followed by
 * mdss_select_accept_sums with the same arguments, with the same outputs value
 * for value (the draw is the same code, run by the row's workgroup once r and the
 * sums are written).  r, the residual sums in accept_workspace, sel_index and
 * sel_token (nullable), out_token, accepted, residual_mass (nullable) and
 * row_status (nullable; SET to the row's flags) as those two calls; u: [B][3] or
 * NULL for Philox(seed, offset + b).  Errors: as the two calls (EUNSUPPORTED for K
 * or s_max out of range, EINVAL for a NULL p, q, r, drafts, out_token or accepted,
 * EWORKSPACE for a workspace under mdss_workspace_bytes_accept(B, V)). */
mdss_status mdss_step_topk_expsum(const float* p, const float* q, const int32_t* drafts, const float* u,
                                  uint64_t seed, uint64_t offset, int64_t B, int64_t V, int32_t K, int32_t s_max,
                                  float* r, int32_t* sel_index, int32_t* sel_token, int32_t* out_token,
                                  uint8_t* accepted, double* residual_mass, int32_t* row_status,
                                  void* accept_workspace, size_t accept_workspace_bytes, void* stream);

/* Bytes of workspace for mdss_induced_dist_pair_expsum and
 * mdss_induced_dist_successive_expsum (0 if the shape is invalid or B = 0). */
size_t mdss_workspace_bytes_pair_expsum(int64_t B, int64_t V);

/* r: [B][V] fp32 out, the induced distribution of X1 ~ q1, X2 ~ q2 (as
 * mdss_induced_dist_pair). */
mdss_status mdss_induced_dist_pair_expsum(const float* p, const float* q1, const float* q2, int64_t B, int64_t V,
                                          float* r, int32_t* row_status, void* workspace, size_t workspace_bytes,
                                          void* stream);

/* r_stages: [K-1][B][V] fp32 out, the stage laws of successive pairwise
 * selection (as mdss_induced_dist_successive), K in [2, MDSS_SUCCESSIVE_MAX_K].
 * workspace: at least mdss_workspace_bytes_pair_expsum(B, V) bytes. */
mdss_status mdss_induced_dist_successive_expsum(const float* p, const float* q, int64_t B, int64_t V, int32_t K,
                                                float* r_stages, int32_t* row_status, void* workspace,
                                                size_t workspace_bytes, void* stream);

/* ---- Truncated alphabet ---------------------------------------------------
 * Section 4 (after the truncated LP): Omega_0 = the m tokens of largest target
 * probability (ties by lower id).  Run any selection and Algorithm 1 with the
 * renormalised target p~ = p 1[Omega_0] / p(Omega_0) in place of p; their output
 * Z has law p~.  mdss_alphabet_post then keeps Z with probability
 * p_a = p(Omega_0) and otherwise draws from the complement of Omega_0 in
 * proportion to p, so the output has law p.  The selection with p~ costs O(m^2)
 * per row on the K = 2 paths (only positive-weight tokens are poles). */

/* p_trunc [B][V] fp32 out: p~ = fp32(p / p(Omega_0)) on Omega_0, 0 elsewhere;
 * mass0 [B] fp64 out: p(Omega_0).  m >= 1 (m >= V keeps every token).  A row with
 * a NaN, infinite or negative entry is flagged MDSS_ROW_BAD_PROB (p_trunc NaN,
 * mass0 NaN).  No workspace. */
mdss_status mdss_truncate_alphabet(const float* p, int64_t B, int64_t V, int32_t m, float* p_trunc, double* mass0,
                                   int32_t* row_status, void* stream);

/* token [B]: Z, the output of Algorithm 1 with target p_trunc (-1 is passed on).
 * Keep Z iff u_keep < mass0 (fp64); else out = the smallest id j with p_trunc(j)
 * = 0 and C_j > u_draw Z_c, C the running sum of p over those tokens in
 * ascending id and Z_c its total (Z_c = 0: keep Z).  u2: [B][2] fp32 (u_keep,
 * u_draw) or NULL: words 0 and 1 of Philox4x32-10 with key = seed and counter
 * (offset + b (low, high word), 0, 1).  out_token [B] int32, kept [B] uint8. */
mdss_status mdss_alphabet_post(const float* p, const float* p_trunc, const double* mass0, const int32_t* token,
                               const float* u2, uint64_t seed, uint64_t offset, int64_t B, int64_t V,
                               int32_t* out_token, uint8_t* kept, void* stream);

/* ---- Optimal acceptance diagnostics ---------------------------------------
 * Theorem 3: for K = 2 drafts from q the best acceptance probability of any
 * token-level selection rule is
 *   P* = min over token sets S of P(S) + Q(S^c)^2 + 2 Q(S) Q(S^c)
 *      = Qt^2 + min_S (P(S) - Q(S)^2)      (P, Q: target / draft mass, Qt = Q(all));
 * Remark 2's K-draft form Qt^K + min_S (P(S) - Q(S)^K) is computed for K > 2
 * (a conjecture of the paper for K > 2, exact for K = 2).  The library
 * evaluates the minimum over the V + 1 prefixes of the tokens ordered by
 * w = p/q ascending (w rounded once to fp32 from the fp64 ratio; q = 0 last;
 * ties by lower token id), which is the minimum over all sets: a minimising set
 * is {w < threshold} by strict convexity of x^K.  O(V) ranking and one scan per
 * row, fp64 sums. */
#define MDSS_OPTIMUM_MAX_K 8

/* Workspace bytes of mdss_optimal_acceptance (0 if the shape is invalid or B = 0). */
size_t mdss_workspace_bytes_optimum(int64_t B, int64_t V);

/* pstar [B] fp64 out: the value above for K in [2, MDSS_OPTIMUM_MAX_K];
 * kstar [B] int32 (nullable): the smallest prefix length of the w order that
 * attains it (0 = the empty set).  A row with a NaN, infinite or negative entry
 * in p or q gets NaN / -1 and MDSS_ROW_BAD_PROB.  workspace: at least
 * mdss_workspace_bytes_optimum(B, V) bytes, 256-byte aligned. */
mdss_status mdss_optimal_acceptance(const float* p, const float* q, int64_t B, int64_t V, int32_t K, double* pstar,
                                    int32_t* kstar, int32_t* row_status, void* workspace, size_t workspace_bytes,
                                    void* stream);

/* Acceptance probability of Algorithm 1 with proposal r against target p:
 * accept[b] = sum_y min(p(y), r(y)) in fp64 (NaN and MDSS_ROW_BAD_PROB for a
 * row with a NaN, infinite or negative entry).  With r from any of the
 * induced-distribution calls, accept / pstar is the fraction of the optimum a
 * selection rule achieves. */
mdss_status mdss_acceptance(const float* p, const float* r, int64_t B, int64_t V, double* accept,
                            int32_t* row_status, void* stream);

/* ---- Truncated linear program (K = 2) -------------------------------------
 * The paper's practical selection rule (Algorithm 2, eq. heur, eq. p_Ieq and
 * the bound eq. p_acc_bnd), for identical drafts (q2 = NULL: both from q1) or
 * drafts from two distributions (X1 ~ q1, X2 ~ q2; non-identical appendix).
 * Ranking: tokens ordered by the key p - q1 q2 (computed in fp64, rounded once
 * to fp32; -0 counts as +0), larger first, ties by lower token id; every
 * token of the vocabulary is ranked.  Omega_1 = the first min(s, V) ranked
 * tokens, Omega_2 = the rest.  For a drafted pair {x, y}, x != y:
 *   both in Omega_2:  tail = MDSS_TLP_SORTED: the earlier-ranked one is selected
 *                     (eq. heur); tail = MDSS_TLP_HALF: each with probability 1/2
 *                     (the sort-free variant, eq. heur2);
 *   one in Omega_1:   that one is selected;
 *   both in Omega_1:  x is selected with probability w[x][y] (either drafting
 *                     order), the weights maximising sum over Omega_1 of
 *                     min(p(k), r(k)) -- the truncated linear program, solved
 *                     exactly (as a maximum flow) on the device.
 * Equal drafts select the first one.  r is the resulting distribution of the
 * selected token (eq. p_Ieq, eq. p_Ieq3 for the HALF tail; the appendix's p~_I
 * for two distributions); it is the proposal of Algorithm 1
 * (mdss_accept_or_resample), and acceptance = sum_y min(p(y), r(y)).
 * At most one LP per position; the SORTED tail sorts each row (O(V) radix
 * passes), the HALF tail only selects the top s. */
#define MDSS_TLP_MAX_S 16
#define MDSS_TLP_SORTED 0
#define MDSS_TLP_HALF 1

/* Workspace bytes of mdss_truncated_lp (0 if the arguments are invalid or B = 0). */
size_t mdss_workspace_bytes_tlp(int64_t B, int64_t V, int32_t tail);

/* p, q1 (and q2 unless NULL): [B][V] fp32 in.  s in [1, MDSS_TLP_MAX_S], tail
 * MDSS_TLP_SORTED or MDSS_TLP_HALF.  Outputs:
 *   r       [B][V] fp32, every entry written;
 *   omega1  [B][s] int32: the Omega_1 tokens in rank order (-1 past min(s, V));
 *   w       [B][s][s] fp64: w[x][y] (x, y < min(s, V), x != y) = probability
 *           that Omega_1 token x is selected from the drafted pair {x, y};
 *           w[y][x] = 1 - w[x][y] as rounded, w[x][x] = 1, other entries 0;
 *           the selection reads only the entries with x < y;
 *   accept  [B] fp64 (nullable): sum_y min(p(y), r(y)), computed from r before
 *           its rounding to fp32.
 * The optimal weights need not be unique; r on Omega_2, omega1 and the
 * optimum value are.  A row with a NaN, infinite or negative entry in p, q1
 * or q2 is flagged MDSS_ROW_BAD_PROB: r and w NaN, omega1 -1, accept NaN.
 * workspace: at least mdss_workspace_bytes_tlp(B, V, tail) bytes, 256-byte
 * aligned. */
mdss_status mdss_truncated_lp(const float* p, const float* q1, const float* q2, int64_t B, int64_t V, int32_t s,
                              int32_t tail, float* r, int32_t* omega1, double* w, double* accept,
                              int32_t* row_status, void* workspace, size_t workspace_bytes, void* stream);

/* Selection between drafts[b][0] ~ q1 and drafts[b][1] ~ q2 (q2 = NULL: q1)
 * under the truncated rule of mdss_truncated_lp, given its omega1 and w for
 * the same p, q1, q2, s and tail: f = Pr(Y = X1 | X1, X2) as above (1 for
 * X1 = X2), index 0 iff u_sel < f (fp64).  A row whose omega1[b][0] is -1 is
 * flagged MDSS_ROW_BAD_PROB; a drafted id outside [0, V) or with q1(X1) = 0 or
 * q2(X2) = 0, MDSS_ROW_BAD_DRAFT; such rows get -1. */
mdss_status mdss_select_truncated_lp(const float* p, const float* q1, const float* q2, const int32_t* drafts,
                                     const float* u, uint64_t seed, uint64_t offset, int64_t B, int64_t V, int32_t s,
                                     int32_t tail, const int32_t* omega1, const double* w, int32_t* sel_index,
                                     int32_t* sel_token, int32_t* row_status, void* stream);

/* Static, thread-safe description of a status code. */
const char* mdss_status_string(mdss_status s);

/* ABI version of this header (incremented on incompatible changes). */
int32_t mdss_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MDSS_H */
