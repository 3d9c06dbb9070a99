/*
 * dd.h - C ABI of the MI355X (gfx950) reverse-step library for discrete-diffusion
 * language models (arXiv 2609.04010, "Unlocking Lossless Speedups in LLMs via
 * Discrete Diffusion").
 *
 * The hot path is one reverse denoising step, run T times:
 *   denoiser   x_theta(z_t, t): a bidirectional pre-LN transformer (Background,
 *              "Discrete Diffusion Language Models": a denoising model maps the
 *              noisy sequence and the time to per-position distributions);
 *   posterior  p_{s|t}(z_s | z_t) = q_{s|t}(z_s | z_t, x = x_theta(z_t, t)),
 *              masked prior (App. A.1, eq. mdm-posterior) with carry-over of
 *              unmasked tokens, or uniform prior (App. A.2,
 *              eq. uniform_true_reverse_posterior);
 *   sample     one categorical draw per position (two-level Gumbel-max).
 *
 * Conventions shared by every entry point
 *   - Pointers documented "device" must be device memory of the current HIP
 *     device; "host" pointers are read during the call only.  The library never
 *     allocates device memory: the caller owns parameters, workspace, logits,
 *     token buffers, noise and traces.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).  Every
 *     compute call is asynchronous and ordered on that stream; nothing
 *     synchronises the host except dd_read_device_error and dd_profile_read.
 *   - Token ids are int32.  V is the number of real tokens (logit width).  For the
 *     masked prior the [MASK] token is id V (the K-th category of the paper's
 *     notation, K = V + 1 classes); for the uniform prior K = V.
 *   - Host-side validation runs before any launch; on failure the call returns
 *     DD_E_ARG / DD_E_SHAPE / DD_E_DTYPE / DD_E_WORKSPACE / DD_E_UNSUPPORTED,
 *     launches nothing and writes no output.  A failed launch returns DD_E_HIP.
 *     dd_last_error() gives a human-readable reason (thread-local).
 *   - Out-of-range token ids met on the device set bit DD_DEVERR_TOKEN in a
 *     device error word (the id is clamped so memory stays in bounds); read it
 *     with dd_read_device_error.  No call aborts and no exception crosses the ABI.
 *   - Tuning override: the environment variable DD_GEMM_TILE = 0..10, when set,
 *     forces one tile variant of the bf16 projections (for tuning and for tests
 *     that cover every variant).  It changes speed and, for the vocabulary
 *     projection, the order in which K-slices are summed; never the operation.
 *     Nothing else in the library reads the environment.
 */
#ifndef DD_H
#define DD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DD_OK = 0,
    DD_E_ARG = 1,         /* null pointer, non-positive size, bad schedule value */
    DD_E_SHAPE = 2,       /* inconsistent shapes (e.g. L > max_len, ld < V)      */
    DD_E_DTYPE = 3,       /* unknown dtype                                       */
    DD_E_WORKSPACE = 4,   /* workspace or parameter buffer too small             */
    DD_E_HIP = 5,         /* a HIP runtime call or launch failed                 */
    DD_E_UNSUPPORTED = 6, /* valid but not implemented (e.g. bf16 with dh != 64) */
    DD_E_DEVICE = 7       /* the device error word is non-zero                   */
} dd_status;

typedef enum { DD_BF16 = 0, DD_FP32 = 1 } dd_dtype;
typedef enum { DD_PRIOR_MASK = 0, DD_PRIOR_UNIFORM = 1 } dd_prior;
typedef enum { DD_NORM_LAYER = 0, DD_NORM_RMS = 1 } dd_norm;

/* Classes per level-1 group of the two-level Gumbel-max draw. */
#define DD_GUMBEL_GROUP 256
/* Device error word bits. */
#define DD_DEVERR_TOKEN 1
#define DD_DEVERR_MASK 2   /* an attention-pattern entry was invalid (see dd_denoise_forward_ex) */
#define DD_DEVERR_LOGITS 4 /* a row's logits gave no valid draw (NaN or +inf, or no finite
                              logit where one is needed); that row's output is a fallback:
                              z_s = z_t (posterior), z = 0 (verification) */

/*
 * Denoiser architecture.  Pre-LN transformer, bidirectional attention (other
 * patterns: dd_denoise_forward_ex):
 *   h = tok_emb[z] + pos_emb[l] + temb(alpha_t)       (temb only if time_cond)
 *   temb_j = sin(tau w_j) (j < d/2), cos(tau w_{j-d/2}) (j >= d/2),
 *   w_i = 10000^(-i/(d/2)), tau = 1000 (1 - alpha_t)
 *   per layer: h += W_o attn(N1(h)) + b_o ; h += W_2 gelu_tanh(W_1 N2(h) + b_1) + b_2
 *   logits = W_out N_f(h)                               (V columns, no bias)
 * The normalisations N (per token row of d features, gain g and shift b from the
 * parameter blob) follow `norm`:
 *   DD_NORM_LAYER  (x - mean) / sqrt(var + eps) g + b, var the biased variance
 *   DD_NORM_RMS    x / sqrt(mean(x^2) + eps) g: RMSNorm over the whole row (the
 *                  paper's own model, Sec. 5.1, uses RMSNorm); the shift vectors
 *                  keep their place in the blob and are not read
 * d_model even, d_model % n_heads == 0.  dtype DD_BF16: bf16 weights and
 * activations, fp32 accumulation, fp32 residual stream, normalisation statistics
 * and softmax; DD_FP32: everything fp32 (validation build).
 *
 * Adapters (lora_rank = r > 0; the diffusion weights of Sec. 3.1, a LoRA
 * adapter on every projection W_qkv, W_o, W_1, W_2): at sequence position l
 * each projection y = W a + b becomes
 *   y = W a + b + g_l (lora_alpha / r) B (A a)
 * with the per-position gate g_l in {0, 1} of dd_denoise_forward_ex (Sec. 3.2,
 * Sec. 4.1: adapters off at clean positions, on at noisy ones; every other
 * entry point runs with all gates on).  g_l = 1 everywhere is the merged weight
 * W + (alpha/r) B A.  r % 8 == 0, lora_alpha > 0; r = 0 disables adapters
 * (lora_alpha is then ignored).
 */
typedef struct {
    int32_t n_layers;
    int32_t d_model;
    int32_t n_heads;
    int32_t d_mlp;
    int32_t vocab;      /* V */
    int32_t mask_id;    /* id of the [MASK] token: V under DD_PRIOR_MASK (the K-th category,
                           Background: Notation), -1 under DD_PRIOR_UNIFORM (no mask);
                           any other value is DD_E_UNSUPPORTED */
    int32_t max_len;    /* rows of the position embedding; L <= max_len */
    int32_t prior;      /* dd_prior: selects tok_emb rows (V + 1 or V) */
    int32_t dtype;      /* dd_dtype of weights, activations and logits */
    int32_t time_cond;  /* 1: add the sinusoidal time embedding */
    int32_t norm;       /* dd_norm: DD_NORM_LAYER or DD_NORM_RMS (other values: DD_E_ARG) */
    float norm_eps;     /* epsilon of the normalisations */
    int32_t lora_rank;  /* r: adapter rank, 0 = no adapters */
    float lora_alpha;   /* adapter scale numerator: scale = lora_alpha / r */
} dd_config;

/* ---------------------------------------------------------------- layout */

/*
 * Parameter blob layout.  Tensor ids in order (every matrix is [out][in],
 * row-major; each tensor starts at a 256-byte aligned offset; element type is
 * cfg->dtype):
 *   0 tok_emb [V+1 or V][d]   1 pos_emb [max_len][d]
 *   per layer l, ids 2 + 12 l + :
 *     0 ln1_g [d]  1 ln1_b [d]  2 w_qkv [3d][d]  3 b_qkv [3d]  4 w_o [d][d]  5 b_o [d]
 *     6 ln2_g [d]  7 ln2_b [d]  8 w_1 [F][d]     9 b_1 [F]    10 w_2 [d][F] 11 b_2 [d]
 *   then lnf_g [d], lnf_b [d], w_out [V][d].
 * With adapters (lora_rank = r > 0) the four projections are stored with r more
 * columns, row o holding W[o][:] then B[o][:] (w_qkv [3d][d+r], w_o [d][d+r],
 * w_1 [F][d+r], w_2 [d][F+r]), and the A matrices follow w_out: per layer l,
 * ids 2 + 12 n_layers + 3 + 4 l + : 0 a_qkv [r][d]  1 a_o [r][d]  2 a_1 [r][d]
 * 3 a_2 [r][F].
 * A vector reports rows = 1, cols = length.
 */
int32_t dd_param_count(const dd_config* cfg);
dd_status dd_param_tensor(const dd_config* cfg, int32_t id, size_t* offset_bytes,
                          int64_t* rows, int64_t* cols);
size_t dd_param_bytes(const dd_config* cfg);

/* Workspace for dd_denoise_forward (activations; the device error word is its
 * first int32).  0 if the configuration is invalid. */
size_t dd_workspace_bytes(const dd_config* cfg, int32_t B, int32_t L);
/* Workspace for dd_sample_loop: the forward workspace plus one logit matrix,
 * the compacted row list with each sequence's first index in it, the per-group
 * log-sum-exps of every logit row and one row log-sum-exp per token row. */
size_t dd_loop_workspace_bytes(const dd_config* cfg, int32_t B, int32_t L);

/*
 * Where dd_sample_loop / dd_psi_sample_loop keep the last reverse step's
 * intermediate values inside their workspace (byte offsets from its start), so
 * that a caller can inspect the arithmetic of a step: run a loop of one step
 * and read these regions once the stream has reached the end of the call.
 *   logits      [rows][logits_ld] of cfg->dtype: the vocabulary projection of the
 *               step.  Compacted (masked prior, bf16, d_model % 128 == 0):
 *               logits row j < *count belongs to token row rows[j]; otherwise
 *               logits row m belongs to token row m.
 *   rows, count int32 [B*L] and int32: the compacted list of the token rows that
 *               were masked before the step and that the step unmasks (stage 0 of
 *               the masked prior's draw: the mask is kept iff the uniform of the
 *               mask's level-1 word is below its probability, which needs no
 *               logits), ascending, and its length; count is
 *               -1 when the loop does not compact.
 *   glse        fp32 [rows][glse_ld]: per-group log-sum-exps of each logits row
 *               (groups of DD_GUMBEL_GROUP classes) when the vocabulary
 *               projection wrote them (see dd_sample_loop), else unspecified.
 *   cand        int32 [rows][glse_ld]: with DD_LOOP_STORE_FREE, each logits row's
 *               per-group candidates (a class id, -1 for a group with no finite
 *               logit); the region is the logits region, which that mode does not
 *               otherwise write.
 *   row_lse     fp32 [B*L]: log-sum-exp over the V logits of every token row the
 *               step drew, in the fp32 arithmetic the draw uses; rows the step
 *               did not draw (carried over) are left as they were.
 * Returns DD_E_ARG for an invalid configuration or B, L <= 0.
 */
typedef struct {
    size_t err, logits, rows, count, glse, cand, row_lse;
    int64_t logits_ld, glse_ld;
} dd_loop_ws_layout;
dd_status dd_loop_workspace_layout(const dd_config* cfg, int32_t B, int32_t L, dd_loop_ws_layout* out);
/* Recommended logit row stride (elements): V rounded up to a multiple of 64. */
int64_t dd_logits_ld(int32_t V);
/* Explicit-noise words per row: level-1 words (one per group, plus one for the
 * mask class under the masked prior: the word of stage 0) followed by one word
 * per real class. */
int32_t dd_noise_width(int32_t prior, int32_t V);

const char* dd_status_str(dd_status s);
const char* dd_last_error(void);

/* Zero the device error word at the start of a workspace (stream-ordered). */
dd_status dd_workspace_reset(void* ws, void* stream);
/* Synchronise `stream`, then copy *err_word (device) to *code_out (host). */
dd_status dd_read_device_error(const int32_t* err_word, int32_t* code_out, void* stream);

/* ---------------------------------------------------------------- compute */

/*
 * dd_init_params - fill the parameter blob (device, `params_bytes` >=
 * dd_param_bytes(cfg)).
 *   host_src == NULL: element e of tensor `id` is a normal drawn by Box-Muller
 *     from Philox4x32-10 block (e>>1 low word, e>>1 high word, id, 3) under key
 *     (seed low, seed high), words 0 and 1 (cosine for even e, sine for odd e);
 *     value 0.02 z (gains: 1 + 0.02 z), computed in float64 and rounded to
 *     nearest-even bf16 / fp32.  (The workloads ask for weights ~ N(0, 0.02).)
 *   host_src != NULL: host blob of dd_param_bytes(cfg) bytes in the layout
 *     above, copied as is.
 */
dd_status dd_init_params(const dd_config* cfg, void* params, size_t params_bytes,
                         uint64_t seed, const void* host_src, void* stream);

/*
 * dd_denoise_forward - logits of x_theta(z_t, t) for B sequences of length L.
 *   z_t     device int32 [B*L], ids in [0, n_tok)
 *   alpha_t schedule value at t (conditions the time embedding), in [0, 1]
 *   logits  device [B*L][ld] of cfg->dtype; columns >= V are left untouched
 *   ld      row stride in elements, ld >= V, ld % 8 == 0
 *   ws      device workspace of >= dd_workspace_bytes(cfg, B, L) bytes
 * Alignment: logits 16 bytes, params and ws 256 bytes (DD_E_ARG otherwise).
 */
dd_status dd_denoise_forward(const dd_config* cfg, const void* params,
                             const int32_t* z_t, int32_t B, int32_t L, double alpha_t,
                             void* logits, int64_t ld, void* ws, size_t ws_bytes,
                             void* stream);

/* Attention patterns (visibility of key j to query i). */
typedef enum {
    DD_ATTN_BIDIRECTIONAL = 0, /* every key (the denoiser's own pattern)                     */
    DD_ATTN_CAUSAL = 1,        /* j <= i: the AR pathway (Sec. 3.1) and the drafting pass over
                                  [context, clean, z_t] (Sec. 4.1)                          */
    DD_ATTN_BLOCK_CAUSAL = 2,  /* blocks of `block` positions: block(j) <= block(i)          */
    DD_ATTN_DRAFT_TRAIN = 3    /* [x, z_1], x and z_1 of L/2 positions in blocks of `block`
                                  (Sec. 3.2, Block Diffusion): causal within x; a token of
                                  noisy block b sees x^(<b) and, causally, its own block     */
} dd_attn_pattern;

/*
 * dd_attn_mask_build - write a pattern in the form the forward pass reads:
 * host int32 out[3*L] = pre[L] | lo[L] | hi[L], key j visible to query i iff
 * j < pre[i] or lo[i] <= j < hi[i].  `block` is used by BLOCK_CAUSAL (>= 1) and
 * DRAFT_TRAIN (>= 1, L even, (L/2) % block == 0); DD_E_ARG / DD_E_SHAPE
 * otherwise.  Host only (no device work).
 */
dd_status dd_attn_mask_build(int32_t pattern, int32_t L, int32_t block, int32_t* out);

/*
 * dd_denoise_forward_ex - dd_denoise_forward with an attention pattern and the
 * per-position adapter gate.
 *   attn_mask  NULL (bidirectional) or device int32 [3*L] in the form of
 *              dd_attn_mask_build, shared by the B sequences.  Needs
 *              0 <= pre <= L, 0 <= lo <= hi <= L and at least one visible key
 *              per query: a query whose entry breaks this sets DD_DEVERR_MASK in
 *              the device error word (first int32 of ws) and sees every key.
 *   lora_gate  NULL (all adapters on) or device int32 [L]: position l uses its
 *              adapters iff lora_gate[l] != 0; shared by the B sequences.
 *              Must be NULL when cfg->lora_rank == 0 (DD_E_ARG).
 * Other arguments, alignment and errors as dd_denoise_forward; the workspace
 * size is dd_workspace_bytes (which accounts for the adapters).
 */
dd_status dd_denoise_forward_ex(const dd_config* cfg, const void* params,
                                const int32_t* z_t, int32_t B, int32_t L, double alpha_t,
                                const int32_t* attn_mask, const int32_t* lora_gate,
                                void* logits, int64_t ld, void* ws, size_t ws_bytes,
                                void* stream);

/*
 * dd_posterior_sample - one reverse-posterior draw per row (App. A.1 / A.2 with
 * x = softmax(logits); App. A.4 eq. psi-sampler at kappa_t = 1).
 *   prior        dd_prior
 *   mask_id      V under DD_PRIOR_MASK (the mask is the K-th category), -1 under
 *                DD_PRIOR_UNIFORM; any other value is DD_E_UNSUPPORTED
 *   logits       device [rows][ld] of logits_dtype (bf16 or fp32), finite or -inf,
 *                at least one finite per read row; ld >= V, ld % 8 == 0.  Under the
 *                masked prior only rows whose z_t is the mask id are read.  A row
 *                that breaks this (NaN, +inf, all -inf) keeps z_s = z_t and sets
 *                DD_DEVERR_LOGITS in dev_err.
 *   z_t          device int32 [rows]; z_s device int32 [rows], may alias z_t
 *   alpha_t, alpha_s  schedule values with 0 <= alpha_t < alpha_s <= 1 (s < t)
 *   noise_words  NULL: Philox4x32-10 noise under key `seed`, counters
 *                (index >> 2, row0 + row, step, 0) for level-1 word `index`
 *                and (class >> 2, row0 + row, step, 1) for the level-2 word of
 *                a class.  Otherwise device uint32 [rows][dd_noise_width] words.
 *                A word w stands for the uniform u = (w + 1/2) 2^-32.
 *   row_lse      NULL, or device fp32 [rows]: for every row that draws (masked
 *                rows under the masked prior, every row under the uniform prior)
 *                the log-sum-exp of its V logits as the draw computes it (fp32,
 *                from the per-group log-sum-exps), so that a caller can form the
 *                draw's probabilities x_v = exp(l_v - row_lse); other rows are
 *                left untouched.
 *   probs        NULL, or device fp32 [rows][K] that receives the posterior
 *                probabilities (debug; a separate float64 kernel; slow).
 *   dev_err      NULL or device int32 error word (DD_DEVERR_TOKEN and
 *                DD_DEVERR_LOGITS are or-ed in).
 * Draw: masked prior, stage 0: the mask class is taken iff u < p_mask, with u =
 * (w + 1/2) 2^-32 of the mask's level-1 word w (compared in double; p_mask =
 * (1 - a_s)/(1 - a_t) needs no logits, App. A.1).  Then, over the real classes,
 * level 1 picks group g by argmax of log M_g + Gumbel (M_g = posterior mass of
 * the group of DD_GUMBEL_GROUP consecutive classes) and level 2 picks the class in
 * g by argmax of log p_j + Gumbel; the lowest index wins ties.  Masked prior: rows
 * with z_t != mask are copied.
 * Arithmetic: log-sum-exp, group masses and Gumbel scores in fp32 (so a draw
 * can differ from an exact one only where two scores lie within ~1e-5); the
 * debug probabilities in float64.
 */
dd_status dd_posterior_sample(int32_t prior, const void* logits, int32_t logits_dtype,
                              int64_t ld, int32_t rows, int32_t V, int32_t mask_id,
                              const int32_t* z_t, double alpha_t, double alpha_s,
                              const uint32_t* noise_words, uint64_t seed, uint32_t step,
                              uint32_t row0, int32_t* z_s, float* row_lse, float* probs,
                              int32_t* dev_err, void* stream);

/*
 * dd_psi_posterior_sample - one Psi-sampler draw per row (App. A.4, eq. psi:
 * kappa q_{s|t} + (1 - kappa) q_s, with x = softmax(logits); closed forms
 * eqs. psi-mdm and psi-usdm).  Arguments as dd_posterior_sample, plus
 *   kappa        correction strength in [0, 1] (DD_E_ARG otherwise); 1 gives
 *                exactly dd_posterior_sample.
 * Masked prior, z_t != mask: x_theta is taken as the one-hot of z_t (the
 * carry-over parameterisation), so the token is kept with probability
 * a_s + kappa (1 - a_s) and remasked otherwise, by stage 0 (remask iff the mask
 * word's uniform is below (1 - kappa)(1 - a_s)); its logits are never read.  Uniform
 * prior: every class keeps non-zero probability for kappa < 1.
 */
dd_status dd_psi_posterior_sample(int32_t prior, const void* logits, int32_t logits_dtype,
                                  int64_t ld, int32_t rows, int32_t V, int32_t mask_id,
                                  const int32_t* z_t, double alpha_t, double alpha_s,
                                  double kappa, const uint32_t* noise_words, uint64_t seed,
                                  uint32_t step, uint32_t row0, int32_t* z_s, float* row_lse,
                                  float* probs, int32_t* dev_err, void* stream);

/*
 * dd_sample_loop - T ancestral steps z_1 -> z_0 on the grid t_k = k/T.
 *   alphas       host double [T + 1], alphas[k] = alpha(k / T): alphas[0] = 1,
 *                alphas[T] = 0 is not required but the values must strictly
 *                decrease in k.
 *   z            device int32 [B*L]; in: z_1, out: z_0
 *   step k = T..1 runs dd_denoise_forward at alphas[k] and dd_posterior_sample
 *   with (alpha_t, alpha_s) = (alphas[k], alphas[k-1]), step = k, row0 = 0 and
 *   noise words noise_words + (k-1) * B*L * dd_noise_width (if non-NULL,
 *   device uint32 [T][B*L][width]) or Philox under `noise_seed`.
 *   z_trace      NULL or device int32 [T + 1][B*L]: z_1 then the state after
 *                each step.
 *   ws           device workspace >= dd_loop_workspace_bytes(cfg, B, L).
 * Masked prior (bf16): each step lists the masked rows that it unmasks (stage 0 of the draw:
 * the mask's probability (1 - a_s)/(1 - a_t), App. A.1, does not depend on the logits) and runs
 * the vocabulary projection and the rest of the draw on those rows only; rows that stay masked
 * and carried-over rows need no logits.  With d_model and d_mlp multiples of 128 and no
 * adapters, the last layer also runs on those rows alone from its attention queries on (keys and
 * values still cover every row), since past that point a row's values reach only its own logits;
 * the listed rows' logits are unchanged.  bf16 with d_model % 128
 * == 0: the vocabulary projection also writes, beside each logit row, the log-sum-exp of each
 * group of DD_GUMBEL_GROUP classes (from the rounded logits it stores), and the draw reads those
 * and one group of logits per row instead of the whole row.  The result equals calling
 * dd_denoise_forward and dd_posterior_sample on every row, up to the summation order inside each
 * group's log-sum-exp (a draw can differ only where two level-1 scores lie within a few ulps);
 * dd_psi_sample_loop with DD_LOOP_POSTERIOR_PASS makes the draw take its own pass over the
 * logit rows instead, as dd_posterior_sample does.  The mask id is cfg->mask_id.  The last
 * step's logits and log-sum-exps stay in the workspace (dd_loop_workspace_layout).
 */
dd_status dd_sample_loop(const dd_config* cfg, const void* params, int32_t B, int32_t L,
                         int32_t T, const double* alphas, int32_t* z,
                         const uint32_t* noise_words, uint64_t noise_seed,
                         int32_t* z_trace, void* ws, size_t ws_bytes, void* stream);

/* dd_psi_sample_loop flags */
#define DD_LOOP_POSTERIOR_PASS 1u /* draw from the posterior's own pass over each logits row
                                     instead of the group log-sum-exps the vocabulary
                                     projection writes (same draws up to summation order) */
#define DD_LOOP_STORE_FREE 2u     /* the store-free draw (masked prior, bf16, d_model % 128 == 0,
                                     Philox noise only): no logits are written.  The vocabulary
                                     projection's epilogue writes, per row and group of
                                     DD_GUMBEL_GROUP classes, the group's log-sum-exp and its
                                     candidate: the first class of the group whose running sum
                                     of exp(logit) exceeds u times the group's sum, u the
                                     uniform of the Philox word (g >> 2, row, step, 5), word
                                     g & 3.  The draw then takes level 1 as always and the chosen
                                     group's candidate as level 2: an exact draw from the same
                                     posterior, with different noise at level 2 (one uniform per
                                     group instead of one Gumbel per class) */

/*
 * dd_psi_sample_loop - dd_sample_loop with the Psi transition (App. A.4,
 * eq. psi-sampler): step k draws with dd_psi_posterior_sample at
 * kappa = kappas[k].
 *   kappas       NULL (every kappa 1: exactly dd_sample_loop) or host double
 *                [T + 1], each used entry (k = 1..T) in [0, 1].
 *   flags        0, DD_LOOP_POSTERIOR_PASS or DD_LOOP_STORE_FREE (both together or
 *                other bits: DD_E_ARG; DD_LOOP_STORE_FREE outside its conditions or
 *                with noise_words: DD_E_UNSUPPORTED).
 * With kappa < 1 decoded tokens can be remasked and T may exceed the number of
 * positions (inference-time scaling, Sec. 4); a step with alpha_s = 1 (the
 * last one) still unmasks every position.  Masked prior (bf16): the rows
 * unmasked before a step first keep or remask (no logits), then the
 * masked rows that the step unmasks run the vocabulary projection and the draw
 * as in dd_sample_loop; the result equals dd_denoise_forward followed by
 * dd_psi_posterior_sample on every row.
 */
dd_status dd_psi_sample_loop(const dd_config* cfg, const void* params, int32_t B, int32_t L,
                             int32_t T, const double* alphas, const double* kappas,
                             uint32_t flags, int32_t* z,
                             const uint32_t* noise_words, uint64_t noise_seed,
                             int32_t* z_trace, void* ws, size_t ws_bytes, void* stream);

/*
 * dd_spec_verify - speculative verification of S drafted blocks (Alg. 1,
 * linear sampler; the rejection correction of speculative decoding).
 *   p_logits     device [S*B][ld] target logits: row s*B + i is p_{i+1} of
 *                sequence s (the last row of a block gives the bonus draw)
 *   q_logits     device [S*(B-1)][ld] draft logits, row s*(B-1) + i is q_{i+1}
 *   draft        device int32 [S][B-1], the drafted tokens x_i (drawn from q_i)
 *   logits_dtype bf16 or fp32; ld >= V, ld % 8 == 0; B >= 1 (q_logits and draft
 *                may be NULL when B == 1)
 *   noise_words  NULL: Philox under `seed` — acceptance uniform u_i from the word
 *                (i >> 2, row0 + s, step, 4), the draw's words as for the
 *                posterior (streams 0 and 1, row row0 + s); otherwise device
 *                uint32 [S][dd_spec_verify_noise_width(B, V)]: B - 1
 *                acceptance words, then the draw's level-1 and level-2 words.
 *   n_out        device int32 [S]: n = the first i (1-based) with
 *                u_i > min(1, p_i(x_i) / q_i(x_i)), or B if none; the block
 *                keeps x_1 .. x_{n-1}
 *   z_out        device int32 [S]: the token that follows them, drawn from
 *                Norm([p_n - q_n]_+) (from p_n if that has no mass) when n < B
 *                and from p_B when n == B, by the two-level Gumbel-max draw
 *   ws           device scratch >= dd_spec_verify_workspace_bytes(S, B) (row
 *                log-sum-exps)
 *   dev_err      NULL or device int32 error word (DD_DEVERR_TOKEN for a draft
 *                token outside [0, V), which is clamped; DD_DEVERR_LOGITS when
 *                the drawn row's logits hold NaN / +inf or no finite value, and
 *                then z_out = 0 for that sequence).
 * Arithmetic in fp32.  Each emitted token is distributed as the target (the
 * tokens per verification forward pass are (n + 1) / 2 with the block's
 * always-accepted first token counted, between 1 and (B + 1) / 2).
 */
size_t dd_spec_verify_workspace_bytes(int32_t S, int32_t B);
int32_t dd_spec_verify_noise_width(int32_t B, int32_t V);
dd_status dd_spec_verify(const void* p_logits, const void* q_logits, int32_t logits_dtype,
                         int64_t ld, int32_t S, int32_t B, int32_t V, const int32_t* draft,
                         const uint32_t* noise_words, uint64_t seed, uint32_t step,
                         uint32_t row0, int32_t* n_out, int32_t* z_out, void* ws,
                         size_t ws_bytes, int32_t* dev_err, void* stream);

/*
 * dd_spec_verify_noalloc - dd_spec_verify for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Same arguments and results as dd_spec_verify, without the
 * workspace: the row log-sum-exps go to a library-held device array of
 * DD_SPEC_VERIFY_NOALLOC_ROWS floats (1 MiB), one per device, which each device
 * the library runs on holds until the process ends.  S (2B - 1) above
 * DD_SPEC_VERIFY_NOALLOC_ROWS is DD_E_WORKSPACE, before any launch.  The call
 * allocates nothing; its first call on a device looks up that device's array
 * (with the device current).  Every call on a device shares the device's array:
 * calls that can overlap on one device (several streams or host threads) race,
 * and the caller must order them.
 */
#define DD_SPEC_VERIFY_NOALLOC_ROWS (1 << 18)
dd_status dd_spec_verify_noalloc(const void* p_logits, const void* q_logits, int32_t logits_dtype,
                                 int64_t ld, int32_t S, int32_t B, int32_t V, const int32_t* draft,
                                 const uint32_t* noise_words, uint64_t seed, uint32_t step,
                                 uint32_t row0, int32_t* n_out, int32_t* z_out, int32_t* dev_err,
                                 void* stream);

/*
 * dd_gaussian_latent_argmax - z = argmax_v (alpha_tilde [v == x] + sigma eps_v)
 * per row (App. A.5: uniform-state diffusion is the argmax projection of a
 * Gaussian diffusion on one-hot vectors).  eps_v = Phi^-1(u) of the Philox word
 * (v >> 2, row0 + row, step, 2) under `seed`; lowest index wins ties.
 *   x      device int32 [rows], ids in [0, V);  z_out device int32 [rows] (may alias x)
 *   alpha_tilde >= 0, sigma > 0 (the workloads use alpha_tilde^2 + sigma^2 = 1)
 */
dd_status dd_gaussian_latent_argmax(const int32_t* x, int32_t rows, int32_t V,
                                    double alpha_tilde, double sigma, uint64_t seed,
                                    uint32_t step, uint32_t row0, int32_t* z_out,
                                    int32_t* dev_err, void* stream);

/* ---------------------------------------------------------------- profiling */

/*
 * Per-launch timing with HIP events on the launching stream.  While enabled,
 * every launch of a kernel class whose bit is set in `class_mask` (bit c =
 * class c; 0 selects every class) gets an event pair: a kernel's pair is
 * recorded by its dispatch (hipExtLaunchKernel), a copy's around the copy.  At
 * most `max_launches` launches are recorded.  For benchmarks.  The recorder is
 * the library's only process-wide mutable state; it is guarded by a mutex, and
 * while it is off (the default) no launch touches it.
 * Classes: 0 time_embedding, 1 embed_layernorm, 2 layernorm, 3 gemm_qkv,
 * 4 attention, 5 gemm_attn_out, 6 gemm_mlp_up, 7 gemm_mlp_down, 8 gemm_vocab,
 * 9 posterior_sample, 10 gaussian_latent, 11 init_params, 12 copy, 13 compact_masked.
 */
dd_status dd_profile_begin(int32_t max_launches, uint32_t class_mask);
dd_status dd_profile_end(void);
int32_t dd_profile_num_classes(void);
/* Synchronises the recorded events; *name is a static string. */
dd_status dd_profile_read(int32_t cls, const char** name, int64_t* launches, double* total_ms);

#ifdef __cplusplus
}
#endif
#endif /* DD_H */
