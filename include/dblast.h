/*
 * dblast.h - C ABI of the DBLast head + stochastic verification library for AMD gfx950.
 *
 * DBLast ("Dependent Block Drafting for Stochastic Speculative Decoding") drafts a block of K
 * tokens from a low-rank latent mixture over R categories,
 *
 *     q(x_1..x_K | y) = sum_z q(z | y) prod_k q_k(x_k | y, z)                 (Eq. cp-drafter)
 *
 * where every branch distribution q_k(. | y, z) is the softmax of the shared target LM head
 * applied to a category-specific hidden state (Sec. "Architecture"), and verifies it against
 * the target with the prefix-marginalised conditional (Eqs. dep-conditional,
 * category-posterior, dep-next-token-distribution) in the sequential accept/residual loop of
 * speculative sampling (Eq. accept-prob; Sec. "Distributional correctness"). This library runs
 * that path on the GPU:
 *
 *   dbl_head_logprobs   branch log-probabilities over the vocabulary (head GEMM + log-softmax)
 *   dbl_sample_block    category and token draw of one block per sequence
 *   dbl_verify_block    sequential accept test, residual or bonus draw, acceptance mass
 *   dbl_expected_len    acceptance mass and expected accepted length along a given trajectory
 *   dbl_acceptance_objective  the training surrogate's forward quantities and the block NLL
 *   dbl_expand_branches / dbl_prior_head  the head's inputs: branch states and category logits
 *   dbl_target_logprobs / dbl_early_determinism  the target side: the sampling transform that
 *                       defines p, and the target-block early-determinism estimate
 *
 * and the same three steps for the greedy-branch proposal that the paper's reported
 * experiments use (appendix "Greedy-Branch Proposal"): dbl_sample_greedy, dbl_verify_greedy,
 * dbl_expected_len_greedy, which take the head's per-row argmax instead of log-probabilities.
 *
 * Notation. B blocks (one per sequence), K drafted positions, R categories, d hidden size, V
 * vocabulary size. The paper writes b for the block length and K for the number of categories.
 * Row m of the branch hidden states and of every per-row output is m = (b*K + k)*R + r, and
 * M = B*K*R. Vocabulary tiles are DBL_VTILE = 128 consecutive ids: tile t holds ids
 * [128 t, min(128 t + 128, V)); nT = ceil(V / 128).
 *
 * Branch log-probabilities are handed over in a two-level form that one pass over V can
 * write without storing logits: for row m and id v in tile t,
 *     lmass[m*nT + t] = log sum_{u in t} exp(logit[m, u])   (tile log-mass)
 *     tls[m*V + v]    = logit[m, v] - lmass[m*nT + t]        (log-prob of v within its tile)
 *     lse[m]          = log sum_u exp(logit[m, u])
 * and every consumer uses the binary32 value  lq(m, v) = fl32(tls + fl32(lmass - lse)).
 *
 * Random draws and discrete decisions follow one determinism contract, so that an
 * independent implementation reproduces every token index bit for bit:
 *  - draws: word 0 of Philox4x32-10 (Salmon et al., SC'11) with counter
 *    (k, purpose, seq mod 2^32, step mod 2^32) and key (seed low 32 bits, seed high 32 bits);
 *    purposes: 0 category, 1 drafted token, 2 accept coin, 3 residual or bonus token;
 *    seq = seq_offset + b (a per-sequence stream);
 *  - probabilities that decide are computed with a deterministic exponential built from
 *    separately rounded IEEE operations (binary32 for token probabilities, binary64 for the
 *    category weights), quantised as floor(p * 2^40) and compared or summed as integers;
 *  - the category posterior is normalised in the log domain with an ascending-z sum; the
 *    mixture at a token is the binary64 sum over ascending z of w_z * q_z;
 *  - an inverse-CDF draw on integer weights W with word r picks the smallest index whose
 *    inclusive cumulative weight exceeds floor(r * sum(W) / 2^32); a position is accepted iff
 *    r * Q < P * 2^32 for the quantised proposal Q and target P at the drafted token.
 *
 * Conventions for every call:
 *  - Ownership: every data pointer is a device pointer owned by the caller; the library never
 *    allocates device memory. Scratch space is a caller-provided device workspace of at least
 *    dbl_workspace_bytes(op, shape) bytes, 256-byte aligned. Every array argument must be
 *    16-byte aligned (the kernels use 16-byte vector loads and stores; any allocator's base
 *    pointer is, a view starting at an element offset may not be); a misaligned one is
 *    DBL_EINVAL.
 *  - Streams: work is enqueued on `stream` (a hipStream_t; NULL is the default stream) and the
 *    call returns without waiting. Outputs are valid once the stream reaches that point. No
 *    call allocates, frees, copies, sets memory or synchronises, and no workspace needs clearing
 *    (within a call, every workspace word is written before it is read), so the calls may be
 *    captured into a HIP graph and replayed.
 *  - Errors: a non-zero dbl_status is returned before anything is launched when an argument is
 *    invalid; DBL_EHIP reports a failed launch. dbl_last_error() gives a message for the
 *    calling thread's last failure. Data-dependent problems (NaN inputs) are not detected.
 *  - Shapes: K, R, d, V >= 1, B >= 0 (B = 0 is a no-op), R <= 64, V < 2^24, d <= 2^20 and
 *    d % 8 == 0 for the bf16 head, M * V < 2^62.
 *  - Thread safety: calls hold no global mutable state apart from the per-thread error text;
 *    concurrent calls on different streams with disjoint outputs and workspaces are safe.
 */
#ifndef DBLAST_H
#define DBLAST_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DBL_VTILE 128

typedef enum {
  DBL_OK = 0,
  DBL_EINVAL = 1,      /* null or misaligned array, negative temperature, bad Kp, ... */
  DBL_ESHAPE = 2,      /* a dimension outside the supported range */
  DBL_EDTYPE = 3,      /* unsupported element type */
  DBL_EWORKSPACE = 4,  /* workspace missing, too small or misaligned */
  DBL_EHIP = 5         /* a HIP runtime call or kernel launch failed */
} dbl_status;

typedef enum { DBL_F32 = 0, DBL_BF16 = 1 } dbl_dtype;

typedef enum {
  DBL_OP_HEAD = 0,
  DBL_OP_SAMPLE = 1,
  DBL_OP_VERIFY = 2,
  DBL_OP_EXPECTED_LEN = 3,
  DBL_OP_SAMPLE_GREEDY = 4,
  DBL_OP_VERIFY_GREEDY = 5,
  DBL_OP_EXPECTED_LEN_GREEDY = 6,
  DBL_OP_TARGET = 7              /* dbl_target_logprobs: rows N = shape.B * shape.K, shape.V */
} dbl_op;

typedef struct {
  int64_t B, K, R, d, V;
} dbl_shape;

/* Tile width of the two-level log-probability form (128). */
int dbl_vtile(void);

/* ceil(V / 128): columns of `lmass`. */
int64_t dbl_ntiles(int64_t V);

/* Workspace bytes needed by `op` at `shape` (0 when the op needs none, SIZE_MAX if invalid). */
size_t dbl_workspace_bytes(int op, dbl_shape shape);

/* Static description of a status code. */
const char* dbl_status_string(int status);

/* Message describing the calling thread's last non-OK status ("" if none). */
const char* dbl_last_error(void);

/*
 * dbl_head_logprobs - branch log-probabilities q_k(. | y, z) for every row (Sec.
 * "Architecture": each branch hidden state goes through the reused target LM head; q is the
 * softmax of the logits).
 *
 *   logit[m, v] = sum_j h[m*d + j] * w[v*d + j],   m < M = B*K*R, v < V
 *
 * in fp32 accumulation, written in the two-level form above; logits are never stored.
 *   dt     DBL_BF16 (bf16 h and w, MFMA path) or DBL_F32 (fp32 h and w)
 *   h      [B, K, R, d] row-major, element type dt: branch hidden states h_{k,z}
 *   w      [V, d] row-major (the lm_head.weight layout; the math weight is w^T), type dt
 *   tls    out [M, V] fp32      lmass  out [M, nT] fp32      lse  out [M] fp32
 *   argmax out [M] int32 or NULL: argmax_v logit[m, v], the lowest id among equal maxima
 *          (the greedy branch tokens x_hat[k, z] of appendix "Greedy-Branch Proposal"); taken on
 *          the same fp32 logits, so tls, lmass and lse are identical with or without it
 *   ws     workspace of dbl_workspace_bytes(DBL_OP_HEAD, shape) bytes (M * 8); needed only
 *          when argmax is requested, otherwise may be 0 and NULL
 * Errors: DBL_EINVAL for null or misaligned pointers, DBL_EDTYPE for other dt, DBL_ESHAPE when
 * d % 8 != 0 (bf16), d > 2^20 or a dimension is out of range, DBL_EWORKSPACE when argmax is
 * requested without workspace.
 */
dbl_status dbl_head_logprobs(dbl_shape shape, int dt, const void* h, const void* w, float* tls,
                             float* lmass, float* lse, int32_t* argmax, void* ws,
                             size_t ws_bytes, void* stream);

/*
 * dbl_sample_block - draw one block per sequence from the latent mixture (Sec. "Dependent
 * Block Drafting and Verification": first a category from the prior, then every position in
 * parallel from that branch). The prior is q_{Z_T}(z) = softmax(prior_logits[b, :] / z_temp)
 * (Sec. "Drafter sampling during inference"); z_temp = 0 selects the highest-prior category
 * (lowest index on ties). Each token x_k ~ q_k(. | z) is drawn in two stages on the head's
 * two-level form: its 128-id tile with probability exp(lmass_t - lse), then the id within the
 * tile with probability exp(tls_v) (their product is q_k(v | z)); each stage is an exact
 * inverse CDF on probabilities quantised to 2^-40, driven by Philox words 0 and 1.
 *   tls, lmass, lse   the head output for this batch (shape.d is unused)
 *   prior_logits      [B, R] fp32 category logits l_z(y)
 *   z_temp            category temperature Z_T >= 0
 *   seed, step        Philox key and step counter; seq_offset + b is block b's sequence index
 *   z_out  out [B] int32 drawn category;  x_out  out [B, K] int32 drafted tokens
 * A row whose quantised probabilities are all zero yields token -1.
 * No workspace (dbl_workspace_bytes(DBL_OP_SAMPLE, .) = 0): ws may be NULL with ws_bytes 0.
 * Errors: DBL_EINVAL for null pointers or z_temp < 0 or NaN; DBL_ESHAPE.
 */
dbl_status dbl_sample_block(dbl_shape shape, const float* tls, const float* lmass,
                            const float* lse, const float* prior_logits, float z_temp,
                            uint64_t seed, uint64_t step, int64_t seq_offset, int32_t* z_out,
                            int32_t* x_out, void* ws, size_t ws_bytes, void* stream);

/*
 * dbl_verify_block - stochastic verification of drafted blocks with the prefix-marginalised
 * conditional q_k(v | x_<k) = sum_z w_{k,z} q_k(v | z), w_{k,z} proportional to
 * q_{Z_T}(z) prod_{j<k} q_j(x_j | z) (Eqs. dep-conditional, category-posterior,
 * dep-next-token-distribution). Position k is accepted with probability
 * min(1, p_k(x_k) / q_k(x_k | x_<k)) (Eq. accept-prob) while all earlier positions were; at
 * the first rejection the replacement is drawn from norm(max(p_k - q_k, 0)) (from p_k itself
 * if that residual has no quantised mass); when all K are accepted and Kp = K + 1 a bonus
 * token is drawn from p_K (Algorithm "Greedy-Branch Dependent Speculative Verification").
 * The verifier does not take the drafted category: it uses the marginal conditional.
 *   x            [B, K] int32 drafted tokens; ids outside [0, V) count as zero-probability
 *   logp         [B, Kp, V] fp32 target log-probabilities p_k(.) (may hold -inf)
 *   Kp           K or K + 1 (the extra row feeds the bonus token)
 *   n_accept     out [B] int32 accepted positions (0..K)
 *   next_token   out [B] int32 residual or bonus token; -1 when all K are accepted and Kp = K
 *   accept_mass  out [B, K] fp32 or NULL: beta_k = sum_v min(p_k(v), q_k(v | x_<k)) along the
 *                draft, every k
 *   al_expected  out [B] fp32 or NULL: AL_b(x) = sum_i prod_{j<=i} A_j (Eq. acceptance-length)
 *   exp_len      out [B] fp32 or NULL: E = sum_i prod_{j<=i} beta_j along the draft
 * Errors: as dbl_sample_block, plus DBL_EINVAL for Kp not in {K, K + 1}.
 */
dbl_status dbl_verify_block(dbl_shape shape, const float* tls, const float* lmass,
                            const float* lse, const float* prior_logits, float z_temp,
                            const int32_t* x, const float* logp, int64_t Kp, uint64_t seed,
                            uint64_t step, int64_t seq_offset, int32_t* n_accept,
                            int32_t* next_token, float* accept_mass, float* al_expected,
                            float* exp_len, void* ws, size_t ws_bytes, void* stream);

/*
 * dbl_verify_block_static - dbl_verify_block for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * arguments without the workspace, the same kernels and bit-identical outputs. Its scratch is a
 * fixed device array inside the library of 8 MiB (8388608 bytes), one copy per GPU, kept until
 * the process ends; the call allocates and frees nothing. Limit: shapes whose verification
 * workspace, dbl_workspace_bytes(DBL_OP_VERIFY, shape), exceeds 8 MiB are rejected (the
 * Qwen3-8B step needs 0.34 MiB, B = 256 blocks of K = 8 at V = 151,936 need 5.0 MiB).
 * Every call on one GPU shares that GPU's array: calls that overlap in time on one GPU (other
 * streams, other threads) race and must not be issued; calls ordered on one stream are safe.
 * `stream` must belong to the current device. Errors: as dbl_verify_block, plus DBL_EWORKSPACE
 * for a shape beyond the fixed scratch and DBL_EINVAL for a stream of another device.
 */
dbl_status dbl_verify_block_static(dbl_shape shape, const float* tls, const float* lmass,
                                   const float* lse, const float* prior_logits, float z_temp,
                                   const int32_t* x, const float* logp, int64_t Kp,
                                   uint64_t seed, uint64_t step, int64_t seq_offset,
                                   int32_t* n_accept, int32_t* next_token, float* accept_mass,
                                   float* al_expected, float* exp_len, void* stream);

/*
 * dbl_expected_len - the expected-accepted-length reduction that the acceptance-oriented
 * objective targets (Sec. "Acceptance-Oriented Training"): along a given trajectory x (for
 * example one drawn from the target), beta_k = sum_v min(p_k(v), q_k(v | x_<k)) with the
 * prefix-marginalised conditional, and E = sum_i prod_{j<=i} beta_j. Forward only.
 *   x       [B, K] int32 conditioning trajectory (ids outside [0, V) count as zero-probability)
 *   logp    [B, K, V] fp32 target log-probabilities
 *   beta    out [B, K] fp32 or NULL;  exp_len  out [B] fp32
 * Errors: as dbl_sample_block.
 */
dbl_status dbl_expected_len(dbl_shape shape, const float* tls, const float* lmass,
                            const float* lse, const float* prior_logits, float z_temp,
                            const int32_t* x, const float* logp, float* beta, float* exp_len,
                            void* ws, size_t ws_bytes, void* stream);

/*
 * Greedy-branch mode (appendix "Greedy-Branch Proposal", "Prefix-Marginalized Conditional",
 * "Distributional Correctness"; Algorithm "Greedy-Branch Dependent Speculative Verification").
 * Each category's branch is decoded greedily, x_hat[b, k, z] = argmax_v q_k(v | y, z) (the
 * argmax output of dbl_head_logprobs, laid out [B, K, R] like the head rows), and the proposal
 * is the mixture of these R deterministic blocks weighted by the prior q_{Z_T}. Verification
 * uses its prefix-marginalised conditional
 *     q(v | x_<k) = sum_{z in C_k} pi~_{k,z} 1{v = x_hat[b, k, z]},
 *     C_k = {z : x_hat[b, j, z] = x_j for all j < k},  pi~_{k,z} = q_{Z_T}(z) / sum_{C_k} q_{Z_T},
 * supported on at most R tokens, so no vocabulary row of the drafter is read. Draws and
 * decisions follow the determinism contract above (pi~ is the log-domain normalisation of the
 * prior restricted to C_k; q at a token is the ascending-z binary64 sum of the matching
 * weights); there is no token draw (purpose 1 is unused). Ids in x_hat outside [0, V) are
 * never proposed tokens.
 */

/*
 * dbl_sample_greedy - draw z ~ q_{Z_T} per block and copy branch z: x[b, k] = x_hat[b, k, z].
 *   x_hat   [B, K, R] int32 branch tokens;  prior_logits [B, R] fp32;  z_temp >= 0
 *   z_out   out [B] int32;  x_out  out [B, K] int32 (-1 for a block whose prior has no
 *           quantised mass)
 * No workspace (dbl_workspace_bytes(DBL_OP_SAMPLE_GREEDY, .) = 0). shape.d is unused.
 * Errors: DBL_EINVAL for null pointers or z_temp < 0 or NaN; DBL_ESHAPE.
 */
dbl_status dbl_sample_greedy(dbl_shape shape, const int32_t* x_hat, const float* prior_logits,
                             float z_temp, uint64_t seed, uint64_t step, int64_t seq_offset,
                             int32_t* z_out, int32_t* x_out, void* stream);

/*
 * dbl_verify_greedy - sequential verification of drafted blocks against the greedy-branch
 * conditional: position k is accepted with probability min(1, p_k(x_k) / q(x_k | x_<k)) while
 * all earlier positions were; the first rejection draws from norm(max(p_k - q(. | x_<k), 0))
 * (from p_k if that has no quantised mass); full acceptance with Kp = K + 1 draws the bonus
 * token from p_K. Arguments and outputs as dbl_verify_block, with x_hat [B, K, R] in place of
 * the log-probability arrays; accept_mass is sum_v min(p_k(v), q(v | x_<k)) over the support.
 * Workspace: dbl_workspace_bytes(DBL_OP_VERIFY_GREEDY, shape) bytes.
 * Errors: as dbl_verify_block.
 */
dbl_status dbl_verify_greedy(dbl_shape shape, const int32_t* x_hat, const float* prior_logits,
                             float z_temp, const int32_t* x, const float* logp, int64_t Kp,
                             uint64_t seed, uint64_t step, int64_t seq_offset, int32_t* n_accept,
                             int32_t* next_token, float* accept_mass, float* al_expected,
                             float* exp_len, void* ws, size_t ws_bytes, void* stream);

/*
 * dbl_expected_len_greedy - beta_k = sum_v min(p_k(v), q(v | x_<k)) with the greedy-branch
 * conditional along a given trajectory x [B, K], and E = sum_i prod_{j<=i} beta_j.
 *   logp [B, K, V] fp32;  beta out [B, K] fp32 or NULL;  exp_len out [B] fp32
 * Workspace: dbl_workspace_bytes(DBL_OP_EXPECTED_LEN_GREEDY, shape) bytes.
 * Errors: as dbl_expected_len.
 */
dbl_status dbl_expected_len_greedy(dbl_shape shape, const int32_t* x_hat,
                                   const float* prior_logits, float z_temp, const int32_t* x,
                                   const float* logp, float* beta, float* exp_len, void* ws,
                                   size_t ws_bytes, void* stream);

/*
 * dbl_acceptance_objective - forward quantities of the acceptance-oriented training surrogate
 * (Sec. "Acceptance-Oriented Training") along target trajectories x* (for example the target's
 * own samples), for the dependent proposal with prior q_{Z_T} = softmax(l / Z_T):
 *   log q(x*_{1:l}) = log sum_z q_{Z_T}(z) prod_{j<=l} q_j(x*_j | z)      (Eq. cp-drafter)
 *   log_r[b, l-1]   = log q(x*_{1:l}) - sum_{j<=l} log p_j(x*_j)  (Eq. acceptance-length-objective)
 *   A_j             = min(1, p_j(x*_j) / q(x*_j | x*_<j)),  q(x_j | x_<j) = q(x_{1:j}) / q(x_{1:j-1})
 *   S[b, l-1]       = sum_{i<=l} prod_{j<=i} A_j
 *   ell_tau[b]      = min({l : r_l < tau} U {K}), 1-based
 *   J[b]            = sum_{l=1}^{ell_tau} (log r_l + log S_l)            (Eq. subblock-objective;
 *                     the training loss is minus its mean, Eq. training-loss)
 *   nll[b]          = -log q(x*_{1:K})                                  (Eq. dependent-nll)
 * Arithmetic is binary64 on the binary32 inputs (lq = fl32(tls + fl32(lmass - lse)) as
 * everywhere); outputs are binary32.
 *   tls, lmass, lse, prior_logits, z_temp   as dbl_expected_len
 *   x       [B, K] int32 trajectory (ids outside [0, V) have probability 0 on both sides)
 *   logp    [B, K, V] fp32 target log-probabilities of the filter that generated x
 *   tau     truncation threshold, finite and > 0 (the paper uses 0.1)
 *   log_r, S  out [B, K] fp32 or NULL;  ell_tau out [B] int32;  J, nll out [B] fp32
 * No workspace. Errors: DBL_EINVAL for null pointers, z_temp < 0 or NaN, tau <= 0 or not
 * finite; DBL_ESHAPE.
 */
dbl_status dbl_acceptance_objective(dbl_shape shape, const float* tls, const float* lmass,
                                    const float* lse, const float* prior_logits, float z_temp,
                                    const int32_t* x, const float* logp, float tau, float* log_r,
                                    float* S, int32_t* ell_tau, float* J, float* nll,
                                    void* stream);

/*
 * dbl_expand_branches - the category hidden expander (Sec. "Architecture"): every trunk state
 * h_k of a block position becomes R branch states
 *     h_{k,z} = h_k + g_z(h_k),   g_z(h) = W_z h + c_z,
 * with the expander a single linear layer H -> R*H (the added parameters of Table 4 besides the
 * prior head). One bf16 MFMA GEMM of the B*K trunk rows against W, fp32 accumulation; the bias
 * and the residual are added in fp32 and the result is rounded once to bf16.
 *   shape   B, K, R, d used (V unused); d % 32 == 0
 *   h       [B, K, d] bf16 trunk states
 *   W       [R*d, d] bf16 (nn.Linear layout; output feature z*d + j is component j of g_z)
 *   c       [R*d] bf16 bias
 *   h_out   out [B, K, R, d] bf16: the dbl_head_logprobs input h
 * No workspace. Errors: DBL_EINVAL for null pointers; DBL_ESHAPE for d % 32 != 0 or a dimension
 * out of range.
 */
dbl_status dbl_expand_branches(dbl_shape shape, const void* h, const void* W, const void* c,
                               void* h_out, void* stream);

/*
 * dbl_prior_head - the category-prior head (Sec. "Architecture"): l[b, z] = U[z] . h_anchor[b]
 * + e[z], the category logits l_z(y) that dbl_sample_block / dbl_verify_block take as
 * prior_logits. fp32 accumulation of bf16 inputs.
 *   shape     B, R, d used;  h_anchor [B, d] bf16 block-anchor states;  U [R, d] bf16;
 *   e         [R] bf16;  prior_logits out [B, R] fp32
 * No workspace. Errors: DBL_EINVAL for null pointers; DBL_ESHAPE.
 */
dbl_status dbl_prior_head(dbl_shape shape, const void* h_anchor, const void* U, const void* e,
                          float* prior_logits, void* stream);

/*
 * dbl_target_logprobs - the target's sampling distribution as log-probabilities, the p of every
 * verification and objective call (Sec. "Acceptance-Oriented Training": the same temperature,
 * top-k and top-p transform generates the trajectories and enters the acceptance probabilities).
 * Per row: s = fl32(logit / T); top-k (k > 0) keeps every id whose s is at least the k-th largest
 * value (ties at the cut are kept); top-p (p < 1) then keeps, visiting the kept ids by decreasing
 * s and increasing id, each id while the integer mass sum floor(detexp32(fl32(s - max)) 2^40) of
 * the ids before it is below ceil(p * total) (binary64 product); log p = s - max - log(sum over
 * kept of exp(s - max)) in binary64, -inf outside the kept set. T = 0 keeps only the lowest-index
 * maximum (log p = 0 there). The kept set is exact and independent of evaluation order.
 *   N, V         rows and vocabulary size (1 <= V < 2^24)
 *   logits       [N, V] fp32 target logits;  logp  out [N, V] fp32, must not overlap logits
 *                (the row is written before the last reads of it)
 *   temperature  finite, >= 0;  top_k  >= 0 (0: off);  top_p  in (0, 1] (1: off)
 *   ws, ws_bytes optional workspace: NULL and 0, or dbl_workspace_bytes(DBL_OP_TARGET, shape)
 *                bytes (256-byte aligned) with shape.B * shape.K = N, shape.V = V. With it, rows
 *                with 0 < top_k <= 256 and V >= 16384 are split over several workgroups
 *                (faster when N is near or below the number of CUs); the output is the same.
 * Errors: DBL_EINVAL for null pointers, overlapping logits and logp, or parameters out of range;
 * DBL_ESHAPE; DBL_EWORKSPACE for a workspace that is too small or misaligned.
 */
dbl_status dbl_target_logprobs(int64_t N, int64_t V, const float* logits, float temperature,
                               int64_t top_k, float top_p, float* logp, void* ws,
                               size_t ws_bytes, void* stream);

/*
 * dbl_early_determinism - target-block early determinism (appendix "Target-Block Early
 * Determinism"): from M blocks x[m] of length b sampled from the target, with p_i the target
 * distribution at position i of block m (row (m*b + i) of logp),
 *     terms[m] = (1/b) sum_{j<=b} prod_{i<=j} p_i(x[m, i]),   mean = (1/M) sum_m terms[m],
 * the estimate of D_b = (1/b) sum_j sum_{u in V^j} p(u)^2. Binary64 accumulation.
 *   x     [M, b] int32 (ids outside [0, V) have probability 0);  logp [M, b, V] fp32
 *   terms out [M] fp32;  mean out scalar fp32 (device) or NULL
 * No workspace. Errors: DBL_EINVAL for null pointers; DBL_ESHAPE.
 */
dbl_status dbl_early_determinism(int64_t M, int64_t b, int64_t V, const int32_t* x,
                                 const float* logp, float* terms, float* mean, void* stream);

/*
 * dbl_stream_read_probe - a diagnostic, not an operation of the method: reads every 16-byte
 * word of buf once (float4 loads, n_partials workgroups of 256 threads striding over the
 * buffer) and writes each workgroup's sum of the values it read to partials[i]. Its time gives
 * the plain streaming-read rate against which the bandwidth-bound kernels are judged.
 *   buf      device, 16-byte aligned, `bytes` bytes (a multiple of 16), read as fp32
 *   partials device, [n_partials] fp32 out;  1 <= n_partials <= 2^20
 * Errors: DBL_EINVAL for null or misaligned pointers; DBL_ESHAPE for sizes.
 */
dbl_status dbl_stream_read_probe(const void* buf, int64_t bytes, float* partials,
                                 int64_t n_partials, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DBLAST_H */
