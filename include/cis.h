/*
 * cis.h — C ABI of the MI355X (gfx950) calibrated-importance-sampling (CIS) token loss.
 *
 * Operation (Yu et al., "Rethinking Training-Inference Mismatch in LLM Reinforcement
 * Learning", arXiv 2609.32444):
 *
 *   For every token row t with training logits z_t[0..V), sampled id y_t, the inference
 *   engine's recorded log-probability l_infer_t (raw, from the sampling step), advantage A_t
 *   and mask m_t:
 *
 *     l_train_t = log softmax(z_t)[y_t]                      (Sec. 3.1: p_t = softmax(z)_y)
 *     k_t       = exp(l_train_t - l_infer_t)                 (Sec. 2.1, Eq. (1): k = p/q)
 *     phi_t     = max(1 - p_t, kappa)                        (Sec. 3.3, Algorithm 1)
 *     w_t       = min{k_t, 1 + lambda * phi_t}               (Eq. (4), Algorithm 1)
 *     term_t    = scale * w_t * A_t * l_train_t
 *     dL/dz_t   = scale * w_t * A_t * (onehot(y_t) - softmax(z_t))
 *
 *   w_t is a stop-gradient constant (Algorithm 1; App. C.1 "Operators"), evaluated from the
 *   difference of the two log-probabilities (the right-hand form of Eq. (4)). lambda is the
 *   paper's threshold: the displacement factor e^eps is truncated at 1 + lambda (Sec. 3.3), so
 *   a bound c on the log-odds displacement itself corresponds to lambda = e^c - 1. kappa is
 *   the numerical floor of Algorithm 1 (5e-3 in the paper). The loss is the REINFORCE form at
 *   update ratio 1, whose gradient is the policy-gradient payload weighted by w_t.
 *
 *   A row is valid when m_t != 0 and 0 <= y_t < V. Invalid rows are not read: l_train, w,
 *   trunc and term are 0 and their gradient row is 0. 1 - p_t is evaluated from the
 *   complement mass sum_{j != y} e^{z_j - max} / sum_j e^{z_j - max}, which keeps its relative
 *   accuracy as p_t -> 1. A token is "truncated" when k_t > 1 + lambda*phi_t (strict).
 *   term_t is 0 when scale*w_t*A_t is 0.
 *
 * Conventions shared by every entry point:
 *   - All array pointers are DEVICE pointers owned by the caller; the library never frees or
 *     retains them and never allocates device memory.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the null stream). The return
 *     value reports argument and launch errors only; it never synchronises. Arguments are
 *     checked before the first launch: on any error other than CIS_ERR_LAUNCH nothing has
 *     been launched and no output has been written. CIS_ERR_LAUNCH means the runtime refused
 *     a launch; kernels queued before it may have run, so the outputs are undefined.
 *   - Data errors (ids out of range on unmasked rows, non-finite rows) are not return codes:
 *     they are counted in the cis_stats_t at the start of the workspace (below).
 *   - The row kernels read a uint8 mask through scalar loads of the aligned 4-byte words that
 *     hold its bytes, so up to 3 bytes before mask[0] and after mask[T-1] are read (and
 *     ignored). Those bytes must be mapped: any hipMalloc allocation or caching-allocator
 *     block (PyTorch's are 512-byte granular) satisfies this; a mask placed within 3 bytes of
 *     the end of a mapped range does not.
 *   - Results are deterministic: repeated calls on the same inputs give identical bits.
 *   - A call issues kernel launches only (no memset or copy operations), so it can be captured
 *     into a HIP graph on `stream` and replayed; a replay reads the buffers as they are then.
 *     The workspace must not be shared by two graphs or calls that may run concurrently.
 */
#ifndef CIS_H
#define CIS_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element type of the logits and of the gradient. */
typedef enum { CIS_BF16 = 0, CIS_F32 = 1 } cis_dtype_t;

/* Status codes. */
enum {
  CIS_OK = 0,
  CIS_ERR_NULL = -1,      /* a required pointer is NULL                                       */
  CIS_ERR_SHAPE = -2,     /* T < 0, V outside [1, 2^28], ld < V or ld_g < V                  */
  CIS_ERR_DTYPE = -3,     /* dtype is not a cis_dtype_t                                       */
  CIS_ERR_PARAM = -4,     /* lambda < 0 or not finite, kappa outside [0,1], scale not finite, */
                          /* an unknown operator or bounds outside their ranges (cis_params_t) */
  CIS_ERR_ALIGN = -5,     /* logits/dlogits base or row stride in bytes not a multiple of 16; */
                          /* workspace not 256-byte aligned                                   */
  CIS_ERR_LAUNCH = -6,    /* the HIP runtime rejected a kernel launch                         */
  CIS_ERR_WORKSPACE = -7, /* workspace smaller than cis_workspace_bytes(T)                    */
  CIS_ERR_ALIAS = -8,     /* dlogits == logits with ld_g != ld, a partial overlap, or an
                             LM-head gradient overlapping an operand or the workspace        */
  CIS_ERR_DEVICE = -9,    /* the current device is not a gfx950 GPU, or no device            */
  CIS_ERR_SCRATCH = -10   /* T > CIS_NOALLOC_MAX_T (cis_loss_bwd_noalloc)                     */
};

/* Per-call statistics, written at byte offset 0 of the workspace by every entry point that
 * takes a workspace, once every row is done (read it after synchronising the stream). The
 * last three fields are the training diagnostics of App. D.1/D.5. */
typedef struct cis_stats {
  double  loss;         /* sum_t term_t, accumulated in double in a fixed order             */
  int64_t n_valid;      /* rows with mask != 0 and 0 <= id < V                              */
  int64_t n_bad_id;     /* rows with mask != 0 and id outside [0, V)                        */
  int64_t n_nonfinite;  /* valid rows whose log-sum-exp is not finite or whose w is NaN     */
  int64_t n_trunc;      /* valid rows the operator acted on ("acted on", App. D.1): for CIS */
                        /* the truncated rows (k > 1 + lambda*phi)                          */
  double  max_abs_logk; /* largest |log k_t| over valid rows (NaN ignored; 0 if none)      */
  double  trunc_excess; /* sum over valid rows of (k_t - w_t) in double, fixed order        */
  int64_t reserved;
} cis_stats_t;

/* Bytes of device workspace cis_loss_fwd/_bwd and cis_weights_ex (without sequence
 * operators) need for T rows (T >= 0). The workspace holds the cis_stats_t, the counters of
 * the fused pass's row queue (which each call clears with a kernel of its own before the rows
 * start) and per-row scratch: loss terms, flags and diagnostics, and for the forward pass the
 * partial sums of up to 32 segments per row (274 bytes per row in all); its previous contents
 * do not matter.
 * Returns 0 for T < 0. */
size_t cis_workspace_bytes(int64_t T);

/* Workspace for the _ex entry points with n_seq responses (n_seq >= 0; pass 0 for token-level
 * operators). Returns 0 for T < 0 or n_seq < 0. */
size_t cis_workspace_bytes_ex(int64_t T, int64_t n_seq);

/* Static, human-readable text for a status code. */
const char* cis_status_string(int status);

/*
 * cis_weights — Algorithm 1 (Sec. 3.3) as one elementwise pass over recorded log-probabilities.
 *
 *   logp_train [T] float  training-side log-probability of each sampled token (<= 0)
 *   logp_infer [T] float  inference-side log-probability recorded at sampling
 *   mask       [T] uint8  nonzero = token counts; NULL = every token counts
 *   lambda, kappa         threshold and floor (lambda >= 0 finite, 0 <= kappa <= 1)
 *   w_out      [T] float  weight min{k, 1 + lambda*max(1-p, kappa)}; 0 on masked tokens
 *   trunc_out  [T] uint8  1 where the cap was applied; NULL = not written
 *
 * Here p = exp(logp_train) and 1 - p is evaluated as -expm1(logp_train).
 * Errors: CIS_ERR_NULL (T > 0 and a required pointer is NULL), CIS_ERR_SHAPE (T < 0),
 * CIS_ERR_PARAM, CIS_ERR_LAUNCH, CIS_ERR_DEVICE.
 */
int cis_weights(const float* logp_train, const float* logp_infer, const uint8_t* mask,
                int64_t T, float lambda, float kappa,
                float* w_out, uint8_t* trunc_out, hipStream_t stream);

/*
 * cis_loss_fwd — the forward pass: training log-softmax at the sampled ids, CIS weights and
 * loss, reading each valid logits row once.
 *
 *   logits     [T, ld] device, dtype elements, row-major; columns [V, ld) are never used.
 *              Base address and ld*sizeof(dtype) must be multiples of 16 bytes.
 *   dtype      CIS_BF16 or CIS_F32
 *   T, V, ld   rows, vocabulary size (1 <= V <= 2^28), row stride in elements (ld >= V);
 *              the buffer spans T*ld elements (the last row's padding included)
 *   ids        [T] int64   sampled token id of each row
 *   logp_infer [T] float   inference log-probability of the sampled id
 *   adv        [T] float   advantage of each row (per-response factors already folded in)
 *   mask       [T] uint8   nonzero = the row counts; NULL = every row counts
 *   lambda, kappa, scale   threshold, floor, and the loss normalisation (e.g. -1/N_valid)
 *   logp_train_out, w_out [T] float, trunc_out [T] uint8, loss_terms_out [T] float:
 *              optional per-row outputs (NULL = not written)
 *   loss_out   [1] float   optional; sum_t term_t rounded to float
 *   workspace  device, 256-byte aligned, >= cis_workspace_bytes(T) bytes; receives cis_stats_t
 * Errors: CIS_ERR_NULL, CIS_ERR_SHAPE, CIS_ERR_DTYPE, CIS_ERR_PARAM, CIS_ERR_ALIGN,
 *         CIS_ERR_WORKSPACE, CIS_ERR_LAUNCH, CIS_ERR_DEVICE.
 */
int cis_loss_fwd(const void* logits, int dtype, int64_t T, int64_t V, int64_t ld,
                 const int64_t* ids, const float* logp_infer, const float* adv,
                 const uint8_t* mask, float lambda, float kappa, float scale,
                 float* logp_train_out, float* w_out, uint8_t* trunc_out,
                 float* loss_terms_out, float* loss_out,
                 void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * cis_loss_bwd — the fused forward and backward pass: everything cis_loss_fwd produces, plus
 * the gradient of sum_t term_t with respect to the logits, written in the logits dtype with
 * round-to-nearest-even.
 *
 *   dlogits    [T, ld_g] device, same dtype as logits; base and ld_g*sizeof(dtype) multiples
 *              of 16 bytes. Columns [V, ld_g) are not written. Every row is written (zeros
 *              for invalid rows). May be the logits buffer itself (in place) when ld_g == ld;
 *              any other overlap is rejected with CIS_ERR_ALIAS.
 *   other arguments as for cis_loss_fwd.
 * Gradient values whose magnitude is below 2^-126 may be flushed to zero.
 */
int cis_loss_bwd(const void* logits, int dtype, int64_t T, int64_t V, int64_t ld,
                 const int64_t* ids, const float* logp_infer, const float* adv,
                 const uint8_t* mask, float lambda, float kappa, float scale,
                 void* dlogits, int64_t ld_g,
                 float* logp_train_out, float* w_out, uint8_t* trunc_out,
                 float* loss_terms_out, float* loss_out,
                 void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Rows per call of cis_loss_bwd_noalloc (the capacity of its fixed scratch). */
#define CIS_NOALLOC_MAX_T 262144

/*
 * cis_loss_bwd_noalloc — cis_loss_bwd for callers that cannot allocate device memory or pass
 * a workspace (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc). Same operation, kernels and results as cis_loss_bwd; the per-row scratch and
 * the cis_stats_t live in a fixed device array of the library (4.5 MiB per device, held until
 * the process ends) instead of a caller's workspace. The call allocates nothing.
 *
 *   T          0 <= T <= CIS_NOALLOC_MAX_T (262144); larger T returns CIS_ERR_SCRATCH before
 *              anything else is checked or launched
 *   stats_out  optional device pointer that receives the call's cis_stats_t (NULL = not
 *              written); the copy kept in the library's array is overwritten by the next call
 *   other arguments as for cis_loss_bwd.
 * Every call on one device uses that device's one array: two calls that may overlap on a
 * device (different streams, or graphs replayed concurrently) race on it and must be
 * serialised by the caller. Nothing in the array needs clearing between calls.
 * Errors: those of cis_loss_bwd except CIS_ERR_WORKSPACE, plus CIS_ERR_SCRATCH; the device
 * check (CIS_ERR_DEVICE) comes before the other argument checks.
 */
int cis_loss_bwd_noalloc(const void* logits, int dtype, int64_t T, int64_t V, int64_t ld,
                         const int64_t* ids, const float* logp_infer, const float* adv,
                         const uint8_t* mask, float lambda, float kappa, float scale,
                         void* dlogits, int64_t ld_g,
                         float* logp_train_out, float* w_out, uint8_t* trunc_out,
                         float* loss_terms_out, float* loss_out, cis_stats_t* stats_out,
                         hipStream_t stream);

/* =========================================================================================
 * The operator family and the decoupled PPO-clip path.
 *
 * The weight on the token loss (App. C.1 "Operators", Table tab:baselines), from the
 * training-side log-probability l_p (probability p) and the inference-side one l_q (q), with
 * k = exp(l_p - l_q). Defaults in parentheses are the paper's hyperparameters.
 *
 *   CIS_OP_CIS        min{k, 1 + lambda*max(1 - p, kappa)}            (Algorithm 1; 2.3, 5e-3)
 *   CIS_OP_NONE       1
 *   CIS_OP_EXACT      k clamped to [lo, hi]                            ([1e-6, 1e6])
 *   CIS_OP_TIS        min(k, hi)                                       (C = hi = 2)
 *   CIS_OP_ICEPOP     k if lo <= k <= hi, else 0                       ([0.5, 5])
 *   CIS_OP_KPOP       k if max(KL_B(p||q), KL_B(q||p)) <= hi, else 0; the Bernoulli KL in
 *                     float64 with p, q clamped to [1e-8, 1 - 1e-8]     (App. D.5; phi = hi = 2)
 *   CIS_OP_TWO_SIDED  max{CIS weight, (1 + p)/2}: the displacement also lifted to e^eps >= 1/2
 *   CIS_OP_QFIXED     min{k, 1/(q + (1 - q)/(1 + lambda))}: a displacement bound
 *                     eps <= log(1 + lambda) mapped to a ratio cap with q held fixed
 *   CIS_OP_SEQ_TIS    min(K, hi) on every token of a response, K = prod of its tokens' k (C = 2)
 *   CIS_OP_SEQ_MIS    K if lo <= K <= hi else 0 on every token of a response ([0.5, 2])
 *
 * Band and clamp edges are inclusive; caps are strict (a token at k = C is not truncated).
 * A token is "acted on" when the operator changed its weight (truncated, masked, clamped or
 * lifted); for the sequence operators, every valid token of an acted-on response. The
 * sequence operators need every token's k before any gradient, so they take l_p from
 * logp_old (the decoupled path) or from cis_weights_ex's logp_p.
 * ========================================================================================= */
typedef enum {
  CIS_OP_CIS = 0,
  CIS_OP_NONE = 1,
  CIS_OP_EXACT = 2,
  CIS_OP_TIS = 3,
  CIS_OP_ICEPOP = 4,
  CIS_OP_KPOP = 5,
  CIS_OP_TWO_SIDED = 6,
  CIS_OP_QFIXED = 7,
  CIS_OP_SEQ_TIS = 8,
  CIS_OP_SEQ_MIS = 9
} cis_op_t;

/* Operator and loss parameters (a host struct, read during the call). */
typedef struct cis_params {
  int32_t op;           /* cis_op_t                                                          */
  float lambda;         /* CIS, two-sided, q-fixed: >= 0, finite                             */
  float kappa;          /* CIS, two-sided: in [0, 1]                                         */
  float lo, hi;         /* EXACT clamp, ICEPOP / SEQ_MIS band (0 <= lo <= hi); TIS / SEQ_TIS */
                        /* cap and KPOP bound (hi >= 0); hi may be +inf                      */
  float clip_low;       /* decoupled path: the update ratio is clipped to                    */
  float clip_high;      /*   [1 - clip_low, 1 + clip_high]; 0 <= clip_low <= 1, clip_high >= 0 */
  float scale;          /* loss normalisation (finite)                                       */
} cis_params_t;

/*
 * cis_weights_ex — the operator family as one pass over recorded log-probabilities.
 *
 *   logp_p [T] float      training-side log-probability of each token (<= 0)
 *   logp_q [T] float      inference-side log-probability recorded at sampling
 *   mask   [T] uint8      nonzero = token counts; NULL = every token counts
 *   seq_offsets [n_seq+1] int64   sequence operators only: response s is the token range
 *                         [seq_offsets[s], seq_offsets[s+1]), rising from 0 to T (tokens
 *                         outside every response get weight 0); NULL / 0 otherwise
 *   params                operator and its bounds (clip_* and scale unused)
 *   w_out     [T] float   weight (0 on masked tokens)
 *   acted_out [T] uint8   1 where the operator acted; NULL = not written
 *   eps_out   [T] float   log-odds displacement logit p - logit q (Sec. 3.1); +inf when only
 *                         p = 1, -inf when only q = 1, log k when both are 1; NULL = not written
 *   workspace             >= cis_workspace_bytes_ex(T, n_seq), 256-byte aligned; receives a
 *                         cis_stats_t (n_valid, n_trunc, max_abs_logk, trunc_excess; loss 0)
 * Here 1 - p is -expm1(logp_p). Errors: CIS_ERR_NULL, CIS_ERR_SHAPE (T < 0, n_seq < 0, or a
 * sequence operator with n_seq < 1 while T > 0), CIS_ERR_PARAM, CIS_ERR_ALIGN,
 * CIS_ERR_WORKSPACE, CIS_ERR_LAUNCH, CIS_ERR_DEVICE.
 */
int cis_weights_ex(const float* logp_p, const float* logp_q, const uint8_t* mask, int64_t T,
                   const int64_t* seq_offsets, int64_t n_seq, const cis_params_t* params,
                   float* w_out, uint8_t* acted_out, float* eps_out,
                   void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * cis_loss_fwd_ex / cis_loss_bwd_ex — the loss of cis_loss_fwd / cis_loss_bwd with any
 * operator, and the decoupled PPO-clip objective of Eq. (1).
 *
 *   logp_old [T] float  NULL: the rate-1 path of cis_loss_fwd, with p from the same logits
 *                       (complement mass), term = scale*w*A*l_train and gradient
 *                       scale*w*A*(onehot - softmax); sequence operators are rejected.
 *                       Non-NULL: the decoupled path (App. C.1). logp_old is the training
 *                       log-probability at the rollout snapshot theta_old; the weight uses
 *                       p = exp(logp_old) (1 - p = -expm1(logp_old)) and the update ratio is
 *                       rho = exp(l_train - logp_old):
 *                         term = scale * w * min(rho*A, clip(rho)*A),
 *                         dL/dz = scale * w * A * rho * (onehot - softmax) where rho*A is the
 *                                 smaller branch (A > 0: rho <= 1 + clip_high; A < 0:
 *                                 rho >= 1 - clip_low; ties unclipped), 0 elsewhere.
 *   seq_offsets, n_seq  as for cis_weights_ex (decoupled path only)
 *   params              operator, bounds, PPO clip and scale
 *   acted_out [T] uint8 1 where the operator acted (the trunc_out of cis_loss_fwd)
 *   eps_out   [T] float per-token displacement as in cis_weights_ex; NULL = not written
 *   workspace           >= cis_workspace_bytes_ex(T, n_seq)
 *   other arguments, outputs and errors as for cis_loss_fwd / cis_loss_bwd, plus
 *   CIS_ERR_PARAM for a sequence operator without logp_old.
 * A row is non-finite when its log-sum-exp is not finite, its weight is NaN, or (decoupled)
 * its update ratio is NaN.
 */
int cis_loss_fwd_ex(const void* logits, int dtype, int64_t T, int64_t V, int64_t ld,
                    const int64_t* ids, const float* logp_infer, const float* logp_old,
                    const float* adv, const uint8_t* mask, const int64_t* seq_offsets,
                    int64_t n_seq, const cis_params_t* params,
                    float* logp_train_out, float* w_out, uint8_t* acted_out,
                    float* loss_terms_out, float* eps_out, float* loss_out,
                    void* workspace, size_t workspace_bytes, hipStream_t stream);

int cis_loss_bwd_ex(const void* logits, int dtype, int64_t T, int64_t V, int64_t ld,
                    const int64_t* ids, const float* logp_infer, const float* logp_old,
                    const float* adv, const uint8_t* mask, const int64_t* seq_offsets,
                    int64_t n_seq, const cis_params_t* params, void* dlogits, int64_t ld_g,
                    float* logp_train_out, float* w_out, uint8_t* acted_out,
                    float* loss_terms_out, float* eps_out, float* loss_out,
                    void* workspace, size_t workspace_bytes, hipStream_t stream);

/* =========================================================================================
 * The loss behind the language-model head: the logits are z_t = W h_t, the output of the
 * policy's final projection (the training engine's logits of Sec. 3.1; App. C.1 trains in
 * bf16), and are never materialised for the whole batch. Rows are processed `chunk` at a time:
 * the chunk's logits are formed in float32 by a matrix-core product, the loss of
 * cis_loss_fwd_ex / cis_loss_bwd_ex is evaluated on them, and the backward forms
 *
 *   dL/dh = G W        and        dL/dW = G^T h,        G = dL/dz  (chunk by chunk),
 *
 * with G rounded to bf16 as the operand of those two products (float32 accumulation).
 *
 * The forward never stores the logits: the product's epilogue reduces each row's float32
 * logits to one (max, exp-sum) pair per 64 columns, and a per-row pass folds them. The
 * backward has two ways to obtain G: by default each chunk's float32 logits are kept in the
 * workspace (one chunk at a time) beside the pairs, and one tiled pass over them writes G and
 * its transpose; with recompute = 1 they are never stored, and the product is formed a second
 * time with an epilogue that writes G (four products instead of three, and
 * 4 * min(T, chunk) * V bytes less workspace).
 * ========================================================================================= */

/* Workspace bytes for cis_lmhead_loss_fwd (with_grad = 0), cis_lmhead_loss_bwd (with_grad = 1)
 * or cis_lmhead_loss_bwd with recompute (with_grad = 2): the loss workspace of
 * cis_workspace_bytes_ex plus, per chunk row, 8 bytes per 64 vocabulary columns and 20 bytes,
 * and the row's float32 logits (with_grad = 1), and with gradients W^T, the
 * chunk's bf16 dL/dz and the transposed operands of one dL/dW group (about 2*V*H + 2*V*chunk +
 * 2*(V + H)*min(T, group) bytes; group as for cis_lmhead_loss_bwd). Returns 0 for T < 0, V
 * outside [1, 2^22], H outside [1, 2^16], chunk outside [1, 2^16], n_seq < 0 or with_grad
 * outside 0..2. */
size_t cis_lmhead_workspace_bytes(int64_t T, int64_t V, int64_t H, int64_t chunk, int64_t n_seq,
                                  int with_grad);

/*
 * cis_lmhead_loss_fwd — the loss (any operator; the decoupled path with logp_old) on the logits
 * hidden * weight^T.
 *
 *   hidden [T, ld_h] bf16   last hidden state of each token row; H <= ld_h <= 2^22, a multiple
 *                           of 8, base 16-byte aligned
 *   weight [V, ld_w] bf16   head weight (row v produces logit v), 1 <= V <= 2^22; H <= ld_w <=
 *                           2^22, a multiple of 8, base 16-byte aligned
 *   chunk                   rows per chunk (1 <= chunk <= 2^16): rows whose logits are formed
 *                           by one product. Results do not depend on chunk.
 *   ids, logp_infer, logp_old, adv, mask, seq_offsets, n_seq, params and the per-row outputs
 *                           as for cis_loss_fwd_ex
 *   workspace               >= cis_lmhead_workspace_bytes(T, V, H, chunk, n_seq, 0), 256-byte
 *                           aligned; receives the cis_stats_t
 * Errors: as for cis_loss_fwd_ex; CIS_ERR_SHAPE also for H or ld_* out of range, CIS_ERR_ALIGN
 * for hidden / weight alignment.
 */
int cis_lmhead_loss_fwd(const void* hidden, int64_t T, int64_t H, int64_t ld_h,
                        const void* weight, int64_t V, int64_t ld_w,
                        const int64_t* ids, const float* logp_infer, const float* logp_old,
                        const float* adv, const uint8_t* mask, const int64_t* seq_offsets,
                        int64_t n_seq, const cis_params_t* params, int64_t chunk,
                        float* logp_train_out, float* w_out, uint8_t* acted_out,
                        float* loss_terms_out, float* eps_out, float* loss_out,
                        void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * cis_lmhead_loss_bwd — everything cis_lmhead_loss_fwd produces, plus the gradients of
 * sum_t term_t with respect to the hidden states and the head weight.
 *
 *   dhidden [T, ld_dh] float32   dL/dh (overwritten; rows of invalid tokens are 0); ld_dh >= H
 *   dweight [V, ld_dw] float32   dL/dW; ld_dw >= H. accumulate_dweight = 0 overwrites it (zeros
 *                                when T = 0), nonzero adds the gradient to its contents. It is
 *                                formed by one product per group of consecutive rows, float32
 *                                partial sums added group by group: a group is
 *                                chunk * floor(16384 / chunk) rows when chunk is a multiple of 8
 *                                below 16384, otherwise chunk rows.
 *   recompute                    0: keep each chunk's float32 logits in the workspace while
 *                                its G is formed (faster); 1: never store them and form the
 *                                logits product twice (less workspace). Results agree to float32
 *                                rounding of the log-sum-exp (not bit for bit).
 *   workspace                    >= cis_lmhead_workspace_bytes(T, V, H, chunk, n_seq,
 *                                1 + recompute)
 * dhidden and dweight must not overlap each other, hidden, weight or the used part of the
 * workspace (CIS_ERR_ALIAS otherwise). recompute outside 0..1 is CIS_ERR_PARAM.
 */
int cis_lmhead_loss_bwd(const void* hidden, int64_t T, int64_t H, int64_t ld_h,
                        const void* weight, int64_t V, int64_t ld_w,
                        const int64_t* ids, const float* logp_infer, const float* logp_old,
                        const float* adv, const uint8_t* mask, const int64_t* seq_offsets,
                        int64_t n_seq, const cis_params_t* params, int64_t chunk,
                        float* dhidden, int64_t ld_dh, float* dweight, int64_t ld_dw,
                        int accumulate_dweight, int recompute,
                        float* logp_train_out, float* w_out, uint8_t* acted_out,
                        float* loss_terms_out, float* eps_out, float* loss_out,
                        void* workspace, size_t workspace_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* CIS_H */
