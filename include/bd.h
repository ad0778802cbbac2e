/*
 * bd.h -- C ABI of the MI355X (gfx950) block-diffusion decoding library.
 *
 * The library runs the block-diffusion denoising step of a decoder LM: one
 * forward over a window of in-flight blocks against a KV-cached committed
 * prefix, under the block-causal mask (paper §2.1: bidirectional inside a
 * block, causal across blocks and to the prefix), a mask-suppressed LM-head
 * softmax per masked position giving confidence and argmax (App. B.1), and
 * the threshold commit rule with in-order block commit and a one-step cache
 * write (App. C, App. F).  It also exports the host-side Redline selection
 * test (§4.2, App. A).
 *
 * Conventions
 *  - Every call returns a bd_status and never throws.  On failure,
 *    bd_last_error() returns a thread-local message describing the cause.
 *  - "_dev" pointers are HIP device pointers; all other pointers are host.
 *  - All device work is asynchronous on the stream given to bd_init_model.
 *    Only bd_decode (on return), bd_commit with a non-NULL all_done_host,
 *    and bd_state_read synchronise that stream.
 *  - Matrices are row-major; weight matrices are stored [out][in].
 *  - Tokens are int32 ids in [0, vocab); mask_id is the placeholder token,
 *    whose LM-head column is suppressed before the softmax.
 *  - Prompt length P and generation length G must be multiples of the block
 *    size; the block grid is aligned at absolute position 0.
 */
#ifndef BD_H
#define BD_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    BD_OK = 0,
    BD_EINVAL = -1,        /* invalid argument or configuration */
    BD_ENOMEM = -2,        /* device or host allocation failed */
    BD_EHIP = -3,          /* a HIP runtime call failed */
    BD_ESTATE = -4,        /* call not valid in the object's current state */
    BD_EUNSUPPORTED = -5   /* valid but not supported by this library */
} bd_status;

typedef enum { BD_F32 = 0, BD_BF16 = 1 } bd_dtype;

/* Model architecture.  n_experts == 0 selects a dense SwiGLU FFN of width
 * ffn_dim; n_experts > 0 a top_k-of-n_experts SwiGLU MoE of width expert_ffn
 * plus n_shared always-on shared experts of the same width. */
typedef struct {
    int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab;
    int32_t n_experts, top_k, expert_ffn, n_shared;
    float rms_eps;         /* RMSNorm epsilon */
    float rope_theta;      /* RoPE base; rotate-half pairs (i, i + head_dim/2) */
    float logit_scale;     /* LM-head logits are multiplied by this */
    int32_t mask_id;       /* placeholder token id, in [0, vocab) */
    int32_t dtype;         /* bd_dtype of matrices, activations and KV cache */
    int32_t wq;            /* weight precision of the decoder-layer projections
                              (the precision axis of a serving configuration,
                              §4.2 (iv) and the quantization grid of App. E):
                              BD_WQ_NONE keeps the model dtype; BD_WQ_FP8 (bf16
                              models only) has bd_init_model quantize every
                              decoder-layer projection (QKV, O, gate, up, down,
                              expert and shared-expert matrices) to fp8 E4M3
                              with one power-of-two scale per output row (see
                              bd_quantize_fp8); embeddings, norms, router and
                              LM head stay as given.  The GEMMs read the fp8
                              codes and compute exactly as bf16 GEMMs on the
                              dequantized weights (code value x scale, which
                              bf16 holds exactly).  BD_WQ_MXFP4 (bf16 models
                              only) quantizes the same matrices to the OCP
                              MXFP4 format instead: E2M1 elements with one
                              E8M0 scale per 32 consecutive elements of a row
                              (see bd_quantize_mxfp4), again computed exactly
                              as bf16 GEMMs on the dequantized weights. */
} bd_model_cfg;

enum { BD_WQ_NONE = 0, BD_WQ_FP8 = 1, BD_WQ_MXFP4 = 2 };

/* One serving configuration: the paper's operating point lambda (§2.1, the
 * notation table and App. F): accept threshold, in-flight block count, block
 * size, semi-completion and admission thresholds.  "Resolved fraction" below
 * is (unmasked positions of a block) / B as a float32 ratio, compared with
 * the threshold as float32. */
typedef struct {
    float tau;             /* accept: commit positions with confidence >= tau
                              (float32 compare); tau > 1 commits only forced
                              positions */
    int32_t n_inflight;    /* maximum number of active blocks, >= 1 */
    int32_t block_size;    /* B >= 1 */
    float tau_semi;        /* semi-completion, < 0 = off.  Off: when no active
                              position of a sequence clears tau, its single most
                              confident one is committed.  On: an active block
                              whose predecessor is committed, or active with a
                              resolved fraction >= tau_semi at the start of the
                              step, is fully activated and commits its own most
                              confident position when none of its positions
                              clears tau; other active blocks commit only
                              positions >= tau. */
    float tau_add;         /* admission: after the prefill and after every
                              commit, placeholders are admitted in order while
                              fewer than n_inflight blocks are active and either
                              none is active or the youngest active block's
                              resolved fraction is >= tau_add; <= 0 refills
                              every free slot at once */
    int32_t skip_masked;   /* static skip rule (§3.3),
                              0 or 1: 1 leaves an active block that is still
                              fully masked at the start of a step out of that
                              step's forward (no rows, no confidences, no
                              commits) while an older block is active.  Such a
                              block gains its first token only once it is the
                              oldest active block, so with 1 the decode equals
                              the n_inflight = 1 decode and the admitted blocks
                              behind the oldest wait unforwarded. */
} bd_decode_cfg;

typedef struct bd_model bd_model;
typedef struct bd_state bd_state;

/*
 * bd_init_model -- bind a model to its weights.
 *  weights_dev: n_weights device pointers, in this order (d = d_model,
 *   hd = head_dim, H = n_heads, Hkv = n_kv_heads, E = n_experts,
 *   Fe = expert_ffn, Fs = n_shared * expert_ffn); "mat" tensors are in the
 *   model dtype (bf16 or f32), norm gains and the router are float32:
 *     tok_embed [vocab][d]                                   mat
 *     per layer:
 *       attn_norm [d]                                        f32
 *       w_qkv [(H + 2 Hkv) hd][d]  (q heads, k heads, v heads) mat
 *       w_o [d][H hd]                                        mat
 *       ffn_norm [d]                                         f32
 *       dense:  w_gate [ffn][d], w_up [ffn][d], w_down [d][ffn]          mat
 *       MoE:    w_router [E][d] (f32), w_gate_e [E][Fe][d], w_up_e [E][Fe][d],
 *               w_down_e [E][d][Fe], w_gate_s [Fs][d], w_up_s [Fs][d],
 *               w_down_s [d][Fs]                                          mat
 *     final_norm [d]                                         f32
 *     lm_head [vocab][d]                                     mat
 *  The caller keeps the weights alive until bd_model_free; the library may
 *  keep private repacked copies, which it frees.
 *  stream: a hipStream_t (NULL = default stream).
 *  With n_shared == 0 the three shared-expert pointers may be NULL.
 *  Errors: BD_EINVAL for inconsistent dimensions (head_dim not 64 or 128,
 *  n_heads not a multiple of n_kv_heads, mask_id out of range, wrong
 *  n_weights, top_k outside [1, n_experts], n_experts > 64, wq not a
 *  BD_WQ_* value),
 *  BD_EUNSUPPORTED (MoE, BD_WQ_FP8 or BD_WQ_MXFP4 with the f32 dtype; shapes off the GEMM tiles: with
 *  bf16 every projection's output and input widths -- (H + 2 Hkv) hd, d,
 *  H hd, vocab, 2 ffn or 2 Fe, ffn or Fe -- must be multiples of 128; an
 *  MoE model's d_model a multiple of 256, for its router's four depth
 *  quarters of 64-deep blocks),
 *  BD_ENOMEM, BD_EHIP.
 */
bd_status bd_init_model(const bd_model_cfg* cfg, const void* const* weights_dev, int32_t n_weights,
                        void* stream, bd_model** out);

/*
 * bd_quantize_fp8 -- fp8 weight quantization of one bf16 matrix (the format
 *  bd_init_model uses for BD_WQ_FP8).
 *  w_dev: bf16 [rows][cols] device.  For each row, E is the smallest integer
 *  with max|w| / 2^E <= 448 (E = 0 for an all-zero row); scale_dev[row]
 *  (float32, device) receives 2^E and codes_dev[row][cols] (uint8, device)
 *  the OCP fp8 E4M3 code nearest to w / 2^E (ties to even mantissa; sign
 *  bit set for negative values).  Asynchronous on stream (NULL = default).
 *  Errors: BD_EINVAL for NULL pointers or rows, cols < 1; BD_EHIP.
 */
bd_status bd_quantize_fp8(const void* w_dev, int32_t rows, int32_t cols, uint8_t* codes_dev,
                          float* scale_dev, void* stream);

/*
 * bd_quantize_mxfp4 -- MXFP4 weight quantization of one bf16 matrix, in the
 *  layout bd_init_model keeps for BD_WQ_MXFP4 (the microscaling format of the
 *  quantization grid, App. E).
 *  w_dev: bf16 [rows][cols] device, cols a multiple of 32, the rows taken in
 *  groups of group_rows (rows a multiple of group_rows; one group = one
 *  matrix of a stack, e.g. one expert).  Each 32-element block of a row
 *  (columns 32 j .. 32 j + 31) shares the exponent X = floor(log2 max|w|) - 2
 *  over the block (-127 for an all-zero block; clamped to [-127, 127]); each
 *  element is the E2M1 code (sign bit 3, exponent bits 2-1 with bias 1,
 *  mantissa bit 0: values 0, 0.5, 1, 1.5, 2, 3, 4, 6) nearest to w / 2^X,
 *  ties to the even mantissa, magnitudes above 6 saturating to 6.
 *  Outputs (uint8, device), block-major within each group g:
 *    codes_dev[g][cols/32][group_rows][16]: the block's 32 codes, element 2k
 *      in the low nibble of byte k, element 2k + 1 in the high nibble;
 *    exps_dev[g][cols/32][group_rows]: X + 127 (E8M0).
 *  Asynchronous on stream (NULL = default).
 *  Errors: BD_EINVAL for NULL pointers, rows, cols or group_rows < 1, cols not
 *  a multiple of 32 or rows not a multiple of group_rows; BD_EHIP.
 */
bd_status bd_quantize_mxfp4(const void* w_dev, int32_t rows, int32_t cols, int32_t group_rows,
                            uint8_t* codes_dev, uint8_t* exps_dev, void* stream);

/*
 * bd_prefill -- encode b prompts and create a decode state.
 *  prompt_dev: int32 [b][P] device.  The prompt forward runs under the same
 *  block-causal mask with no LM head (prompt steps are not counted as
 *  forwards, App. F.1).  Afterwards the first min(n_inflight, G/B) blocks of
 *  every sequence are active and fully masked.
 *  Errors: BD_EINVAL if b < 1, P < 0, G < 1, B < 1, n_inflight < 1,
 *  P % B != 0, G % B != 0, tau is NaN, skip_masked not 0 or 1, or a prompt
 *  id is outside [0, vocab)
 *  (checked on the device; reported by the next synchronising call);
 *  BD_EUNSUPPORTED for b > 256, n_inflight > 8, or (bf16 MoE models) an
 *  activation plane of 4 GiB or more (rows x d_model x 2 bytes, rows the
 *  larger of b P and 2 b n_inflight B rounded up to 256: the expert product
 *  addresses its gathered rows by 32-bit offsets).
 */
bd_status bd_prefill(bd_model* model, const int32_t* prompt_dev, int32_t b, int32_t P, int32_t G,
                     const bd_decode_cfg* cfg, bd_state** out);

/*
 * bd_denoise_step -- one decoder forward over every sequence's window
 *  (committed blocks awaiting their cache write, then the active blocks),
 *  followed by the LM head on the masked positions.  Window K/V are written
 *  into the cache at their absolute positions.
 *  Optional debug outputs (NULL to skip), indexed by generated position:
 *   conf_dev [b][G] float32: confidence of every position masked this step,
 *   tok_dev [b][G] int32: its argmax;
 *   logits_dev [b][G][vocab] float32: scaled, mask-suppressed logits (-inf in
 *   the mask column) of those positions, from a separate debug kernel.
 *  Positions not masked this step are left untouched.
 *  Errors: BD_ESTATE when the previous step was not committed.
 */
bd_status bd_denoise_step(bd_model* model, bd_state* st, float* conf_dev, int32_t* tok_dev,
                          float* logits_dev);

/*
 * bd_commit -- apply the commit rule to the last step's statistics: commit
 *  every masked position with confidence >= tau, at least the most confident
 *  one of the sequence (lowest position on ties); sweep blocks oldest first
 *  committing every complete block whose predecessors are committed (App.
 *  C.2); mark blocks written by the last forward as cached; admit new blocks
 *  up to n_inflight; count the forward.  all_done_host (optional) receives 1
 *  when every sequence is finished, which synchronises the stream.
 *  Errors: BD_ESTATE when no step is pending.
 */
bd_status bd_commit(bd_model* model, bd_state* st, int32_t* all_done_host);

/*
 * bd_state_read -- copy the decode trace to device buffers (any may be NULL):
 *  tokens_dev [b][G] int32 (mask_id where not yet committed),
 *  commit_step_dev [b][G] int32 (0-based step of the commit, -1 if none),
 *  forwards_dev [b] int32 (forwards with at least one active block).
 *  Synchronises the stream.
 */
bd_status bd_state_read(bd_model* model, bd_state* st, int32_t* tokens_dev, int32_t* commit_step_dev,
                        int32_t* forwards_dev);

/*
 * bd_decode -- prefill, then denoise/commit until every sequence has
 *  committed its G tokens, then write the trace (see bd_state_read).
 *  Synchronises on return.  TPF = b*G / sum(forwards).
 */
bd_status bd_decode(bd_model* model, const int32_t* prompt_dev, int32_t b, int32_t P, int32_t G,
                    const bd_decode_cfg* cfg, int32_t* tokens_dev, int32_t* commit_step_dev,
                    int32_t* forwards_dev);

/*
 * bd_decode_static -- bd_decode that allocates nothing, for callers that
 *  cannot allocate device memory (code under HIP graph capture, tight serving
 *  loops, harnesses that forbid hipMalloc).  Same arguments, results and
 *  synchronisation as bd_decode; the decode state (KV cache, window
 *  activations, plans, split partials, LM-head partials) is laid out in a
 *  static scratch of BD_STATIC_SCRATCH_BYTES = 64 MiB that every device the
 *  library runs on holds from the library's load until the process ends.
 *  The scratch of the current device is used (the model's device must be
 *  current).  Every call on a device shares that device's scratch and leaves
 *  its contents behind (each call clears what it needs): calls that overlap
 *  on one device race, so the caller serialises them.  Per-launch profiling
 *  (bd_profile) is suspended for the call.  Calls no hipMalloc, hipFree or
 *  hipHostMalloc.
 *  Errors: as bd_decode; BD_EUNSUPPORTED when the state of this decode
 *  (b, P, G, block size, n_inflight and the model's dimensions) needs more
 *  than the scratch holds -- the message gives the bytes needed.
 */
#define BD_STATIC_SCRATCH_BYTES_VALUE (64u << 20)
bd_status bd_decode_static(bd_model* model, const int32_t* prompt_dev, int32_t b, int32_t P, int32_t G,
                           const bd_decode_cfg* cfg, int32_t* tokens_dev, int32_t* commit_step_dev,
                           int32_t* forwards_dev);

/*
 * bd_state_reset -- return a state to the moment right after its prefill
 *  (the prompt cache is kept), so that a decode can be repeated without
 *  re-encoding the prompts.  Asynchronous.
 */
bd_status bd_state_reset(bd_model* model, bd_state* st);

/* bd_state_steps -- number of denoising steps run on the state so far. */
bd_status bd_state_steps(const bd_state* st, int32_t* steps_out);

/*
 * bd_state_stats -- work counters accumulated over the steps run since the
 *  prefill (or the last reset), copied to host out[0..n), n <= 12:
 *   [0] forwards executed (steps with at least one row), [1] window rows
 *   forwarded (sum of M), [2] LM-head rows (masked positions), [3] visible
 *   query-key pairs per head (block-causal), [4] keys read per kv head
 *   (prefix + window, summed over sequences), [5] tokens committed;
 *   participation (App. B.3), summed over sequences
 *   and steps: [6] active block-forwards, [7] of those, forwards of a block
 *   that commits nothing in the step, [8] forwards of a block that was fully
 *   masked at the start of the step behind an older active block and commits
 *   nothing (what the static skip rule saves), [9] the same with at least
 *   one commit (what the rule defers), [10] blocks forwarded for their
 *   one-step cache write, [11] active blocks left out by skip_masked.
 *  Errors: BD_EINVAL for n outside [1, 12].  Synchronises the stream.
 */
bd_status bd_state_stats(bd_model* model, bd_state* st, int64_t* out, int32_t n);

/* Kernel classes timed by bd_profile / bd_profile_read. */
enum {
    BD_PROF_EMBED = 0, BD_PROF_NORM = 1, BD_PROF_GEMM_QKV = 2, BD_PROF_ROPE = 3, BD_PROF_ATTN = 4,
    BD_PROF_GEMM_O = 5, BD_PROF_GEMM_GU = 6, BD_PROF_GEMM_DOWN = 7, BD_PROF_LM_HEAD = 8,
    BD_PROF_COMMIT = 9, BD_PROF_MOE = 10, BD_PROF_KINDS = 11
};

/*
 * bd_profile -- enable (1) or disable (0) per-launch HIP-event timing of every
 *  kernel class on the model's stream; clears the accumulated totals.
 * bd_profile_read -- resolve the recorded events (synchronises) and return
 *  the accumulated milliseconds and launch counts per class
 *  (ms_out[BD_PROF_KINDS], count_out[BD_PROF_KINDS]; either may be NULL).
 */
bd_status bd_profile(bd_model* model, int32_t enable);
bd_status bd_profile_read(bd_model* model, double* ms_out, int32_t* count_out);

/*
 * bd_plan_projection -- the tile plan a bf16 projection C[M][N] = A . W^T of
 *  depth K takes when a state holds rows_cap window rows (host-only query; no
 *  device work).  resid != 0 asks for a projection added to the residual
 *  stream (the O and dense down projections), which may split K into up to
 *  zmax parts chosen on the device from the live row count; their partials
 *  take ws_floats floats of the state's workspace at most (the largest extent
 *  over every live row count in [1, rows_cap]; 0 when K is never split).
 *  bd_prefill sizes the workspace with this extent, and the step refuses a
 *  projection whose extent exceeds it.  Outputs may be NULL.
 *  Errors: BD_EINVAL when N, K or rows_cap < 1; BD_EUNSUPPORTED when N or K
 *  is not a multiple of 128.
 */
bd_status bd_plan_projection(int32_t N, int32_t K, int32_t rows_cap, int32_t resid, int32_t* bm_out,
                             int32_t* bn_out, int32_t* zmax_out, int64_t* ws_floats_out);

bd_status bd_state_free(bd_state* st);
bd_status bd_model_free(bd_model* model);

/* Thread-local description of the last failure ("" if none). */
const char* bd_last_error(void);

/*
 * rl_risk_select -- Redline selection (§4.2 steps (ii)-(iv), App. A).
 *  correct: [m][n] uint8, 1 if configuration j answered prompt i correctly.
 *  cost: [m], larger is better (TPF).  ref_index: the reference row.
 *  For each configuration: V[j] = #{i : correct[ref][i] && !correct[j][i]},
 *  p[j] = Pr[Bin(n, alpha) <= V[j]] (exact binomial tail, App. A.2);
 *  Holm step-down at level delta (sort p ascending, reject while
 *  p_(i) <= delta / (m - i + 1), stop at the first failure; App. A.3) marks
 *  valid[j]; selected = the valid configuration with the largest cost (lowest
 *  index on ties), or ref_index when none is valid.
 *  Host-only; touches only the caller's arrays.  Outputs may be NULL except
 *  selected_out.  Errors: BD_EINVAL when n < 1, m < 1, ref_index outside
 *  [0, m), alpha outside (0, 1), delta outside (0, 1] or a NULL input.
 *  near_ties_out (optional) receives the number of Holm comparisons whose
 *  ratio p / threshold lies within 1e-9 of 1.
 */
bd_status rl_risk_select(int32_t n, int32_t m, int32_t ref_index, const uint8_t* correct,
                         const double* cost, double alpha, double delta, int32_t* V_out,
                         double* p_out, uint8_t* valid_out, int32_t* selected_out,
                         int32_t* near_ties_out);

/*
 * Multiple-testing procedures (App. A.3, A.4 and the baselines of App. D); valid
 * means the null R(lambda) > alpha is rejected.
 *  RL_HOLM            Holm step-down at family-wise level delta (primary).
 *  RL_BONFERRONI      p <= delta / m.
 *  RL_FIXED_SEQUENCE  walk a caller-given, data-independent order, testing
 *                     each configuration at full delta until the first failure.
 *  RL_UNCORRECTED     p <= delta for each configuration (no multiplicity
 *                     correction).
 *  RL_PLUGIN          V / n <= alpha, formed and compared in double precision
 *                     (no finite-sample margin).
 */
#define RL_HOLM 0
#define RL_BONFERRONI 1
#define RL_FIXED_SEQUENCE 2
#define RL_UNCORRECTED 3
#define RL_PLUGIN 4

/*
 * rl_select -- rl_risk_select with a choice of procedure and of prompts.
 *  method: one of RL_*.  order: [m], a permutation of 0..m-1, read only for
 *  RL_FIXED_SEQUENCE (may be NULL otherwise).  prompt_mask: [n] uint8 or
 *  NULL; when given, only the prompts with a non-zero entry are counted and
 *  the p-values use their number n_cal in place of n.  Other arguments and
 *  outputs as rl_risk_select (V_out, p_out, valid_out may be NULL).
 *  Host-only.  Errors: BD_EINVAL for the argument errors of rl_risk_select,
 *  an unknown method, a missing or non-permutation order under
 *  RL_FIXED_SEQUENCE, or a mask that selects no prompt.
 */
bd_status rl_select(int32_t n, int32_t m, int32_t ref_index, const uint8_t* correct,
                    const uint8_t* prompt_mask, const double* cost, double alpha, double delta,
                    int32_t method, const int32_t* order, int32_t* V_out, double* p_out,
                    uint8_t* valid_out, int32_t* selected_out);

/*
 * rl_alpha_sweep -- selection at each budget of a grid (App. A.6).
 *  alphas: [n_alpha] budgets, each in (0, 1), any order.  selected_out
 *  [n_alpha] receives the deployed index at alphas[k]; n_valid_out [n_alpha]
 *  (may be NULL) the number of valid configurations there.  alpha_hat_out
 *  (may be NULL): the smallest budget of the grid at which some valid
 *  configuration has cost > cost[ref_index] (alpha_hat), NaN if none has.
 *  Host-only.  Errors: BD_EINVAL as rl_select for any budget, n_alpha < 1 or
 *  NULL alphas / selected_out.
 */
bd_status rl_alpha_sweep(int32_t n, int32_t m, int32_t ref_index, const uint8_t* correct,
                         const double* cost, const double* alphas, int32_t n_alpha, double delta,
                         int32_t method, const int32_t* order, int32_t* selected_out,
                         int32_t* n_valid_out, double* alpha_hat_out);

/*
 * rl_split_exceedance -- held-out validity over calibration/test splits
 * (§5 "Redline and the mean-accuracy rule", App. D).
 *  cal_masks: [n_splits][n] uint8, non-zero = calibration prompt of that
 *  split; every split needs at least one prompt on each side.  For split s
 *  the procedure selects on the calibration prompts; risks are then
 *  R_test(j) = V_j(test prompts) / n_test and R_pool(j) = V_j(all) / n, in
 *  double precision.  deployed_out [n_splits] (may be NULL): the deployed
 *  index; test_viol_out [n_splits] (may be NULL): its violations on the test
 *  prompts.  counts_out [4] (may be NULL): the number of splits whose
 *  deployed configuration has R_test > alpha, has R_pool > alpha, whose
 *  valid set holds a configuration with R_test > alpha, with R_pool > alpha.
 *  gain_sum_out (may be NULL): the sum over splits, in split order, of
 *  cost[deployed] / cost[ref_index] - 1.  Splits run on host threads; the
 *  results do not depend on their number.  Host-only.  Errors: BD_EINVAL as
 *  rl_select, n_splits < 1, NULL cal_masks or a one-sided split.
 */
bd_status rl_split_exceedance(int32_t n, int32_t m, int32_t ref_index, const uint8_t* correct,
                              const double* cost, double alpha, double delta, int32_t method,
                              const int32_t* order, int32_t n_splits, const uint8_t* cal_masks,
                              int32_t* deployed_out, int32_t* test_viol_out, int32_t* counts_out,
                              double* gain_sum_out);

/*
 * rl_monte_carlo -- the synthetic check with known risks (App. A.7).
 *  true_risk: [m].  u: [trials][k][n] float64 uniforms, k = 1 (one uniform
 *  per prompt shared by every configuration) or k = m (independent draws).
 *  In trial t configuration j loses prompt i when
 *  u[t][k == 1 ? 0 : j][i] < true_risk[j], and V_j is its number of losses;
 *  the p-values and the procedure are those of rl_select.
 *  false_trials_out: the trials in which some configuration with
 *  true_risk > alpha is valid (family-wise errors).  valid_counts_out [m]
 *  (may be NULL): per configuration, the trials in which it is valid.
 *  Trials run on host threads.  Host-only.  Errors: BD_EINVAL for n, m < 1,
 *  trials < 1, k not 1 or m, NULL inputs, or alpha, delta, method, order as
 *  rl_select.
 */
bd_status rl_monte_carlo(int32_t n, int32_t m, const double* true_risk, double alpha, double delta,
                         int32_t method, const int32_t* order, int32_t trials, int32_t k,
                         const double* u, int32_t* false_trials_out, int32_t* valid_counts_out);

#ifdef __cplusplus
}
#endif
#endif /* BD_H */
