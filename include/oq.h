/*
 * oq.h -- C ABI of liboq.so, the MI355X (gfx950) implementation of
 * OmniQuant's block-wise calibration step (arXiv 2308.13137).
 *
 * Conventions shared by every entry point
 *   - Tensors are caller-owned, contiguous, row-major DEVICE pointers,
 *     16-byte aligned.  Nothing is retained after a call returns.
 *   - Every call is asynchronous on the given stream (NULL = the default
 *     stream) and is stateless; calls on different streams may overlap.
 *   - Output buffers are overwritten, never accumulated into.
 *   - Results are deterministic: no atomics, fixed reduction orders; two
 *     identical calls produce identical bytes.
 *   - Arguments are validated before anything is launched.  On error nothing
 *     is launched, the status says why and oq_last_error() (thread-local)
 *     holds a readable detail string.  A failed HIP launch returns OQ_ERR_HIP.
 *   - Optional pointers may be NULL: s = NULL means ones, delta = NULL
 *     zeros, B = NULL no bias, any optional output NULL means "not wanted".
 *   - Supported quantisation: bits in [2, 8] (weights) and [2, 8] or 16
 *     (activations, 16 = not quantised); group g divides C_in and is a
 *     power of two in [8, 512] or equal to C_in (per output channel);
 *     C_in, T and every leading dimension are multiples of 8.
 *   - Entry points that need scratch memory take a caller workspace and a
 *     matching *_workspace_size query.
 *
 * Numerics fixed for all kernels (identical integer codes to any
 * implementation that follows the same order): every named quantity is one
 * IEEE fp32 rounding, no fused multiply-add, round half to even, correctly
 * rounded division and square root; clip strengths are the fp64 sigmoid of
 * their logits rounded once to fp32.  Quantiser, per group of g weights w~:
 *     gamma = sigmoid(gamma_logit), beta = sigmoid(beta_logit)
 *     a = gamma*max, b = beta*min, h = max((a - b)/(2^N - 1), 1e-5)
 *     r = 1/h, z = -rint(b*r), code = clamp(rint(w~*r) + z, 0, 2^N - 1)
 *     w_hat = (code - z)*h
 * max/min ties resolve to the lowest index.  Backward passes use the
 * straight-through estimator: only rint has derivative 1; clamp, max/min and
 * the 1e-5 guard are differentiated exactly.
 */
#ifndef OQ_H
#define OQ_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  OQ_OK = 0,
  OQ_ERR_INVALID_ARG = 1,   /* NULL required pointer, bad shape or stride  */
  OQ_ERR_UNSUPPORTED = 2,   /* valid request outside the supported set     */
  OQ_ERR_WORKSPACE = 3,     /* workspace NULL or smaller than the query    */
  OQ_ERR_HIP = 4            /* a HIP call or launch failed                 */
} oq_status;

typedef enum { OQ_F32 = 0, OQ_BF16 = 1 } oq_dtype;

/* Weight quantisers (the appendix compares LWC with PACT and LSQ run in its
 * place inside the same pipeline, weight clipping only).  Each has two
 * parameters per group, p1 and p2:
 *   OQ_WQ_LWC   clip-strength logits (gamma_logit, beta_logit), Eq. 2
 *   OQ_WQ_PACT  the grid's upper and lower thresholds (hi, lo) learned
 *               directly: a = hi, b = lo in Eq. 2's order; PACT's
 *               straight-through rule (identity on the clipped weight):
 *               d hi = sum of dW^ over codes saturated at 2^N - 1,
 *               d lo = over codes saturated at 0, dW~ = dW^ * [in range]
 *   OQ_WQ_LSQ   step h and zero point z learned directly (h floored at
 *               1e-5, z rounded in the forward); rint has derivative 1 on
 *               codes and zero point; LSQ's gradient scale 1/sqrt(g (2^N-1))
 *               multiplies both: d h = gs * sum dW^((q - z) - m w~/h),
 *               d z = -gs * h * sum dW^(1 - m), dW~ = dW^ * m
 * Activation quantisation by default is per-token asymmetric MinMax; OR-ing
 * OQ_ACT_SYM into an activation bit width (2..8) selects symmetric absmax:
 * h = max(max|x~| / (2^(N-1) - 1), 1e-5), zero point 2^(N-1), codes
 * clamp(rint(x~/h) + 2^(N-1), 0, 2^N - 1); the gradient of max|x~| goes to
 * the lowest index holding it, with that element's sign. */
#define OQ_WQ_LWC 0
#define OQ_WQ_PACT 1
#define OQ_WQ_LSQ 2
#define OQ_ACT_SYM 0x100

const char* oq_status_str(oq_status s);
const char* oq_last_error(void);
int oq_version(void);

/* ---------------------------------------------------------------------------
 * Learnable weight clipping, forward (Sec. 3.2, Eq. 2).
 *   W            [c_out, c_in] (w_dt)      frozen full-precision weight
 *   s            [c_in] fp32 | NULL        LET scale: quantises W~ = s (.) W (Eq. 3)
 *   gamma_logit,
 *   beta_logit   [c_out, c_in/group] fp32  clip-strength logits, one pair per group;
 *                                          a group is `group` consecutive input
 *                                          channels of one output row
 *   W_dq         [c_out, c_in] (dq_dt) | NULL   dequantised weight (code - z)*h
 *   codes        [c_out, c_in] uint8 | NULL     integer codes in [0, 2^bits - 1]
 *   h, z         [c_out, c_in/group] fp32 | NULL   step and (integer-valued) zero point
 */
oq_status oq_lwc_fakequant_fwd(const void* W, oq_dtype w_dt, int64_t c_out, int64_t c_in,
                               const float* s, const float* gamma_logit, const float* beta_logit,
                               int bits, int64_t group, void* W_dq, oq_dtype dq_dt,
                               uint8_t* codes, float* h, float* z, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Learnable weight clipping, straight-through backward (Sec. 3.2, Eq. 2).
 *   dW_dq          [c_out, c_in] fp32   dL/d(dequantised weight)
 *   d_gamma_logit,
 *   d_beta_logit   [c_out, c_in/group] fp32 (required)
 *   d_s            [c_in] fp32 | NULL   weight-path part of dL/ds: sum_o dL/dW~[o,c] * W[o,c]
 *   dW_tilde       [c_out, c_in] fp32 | NULL   dL/dW~ per element
 * Workspace: oq_lwc_fakequant_bwd_workspace_size (0 bytes when d_s is NULL).
 */
oq_status oq_lwc_fakequant_bwd(const void* W, oq_dtype w_dt, int64_t c_out, int64_t c_in,
                               const float* s, const float* gamma_logit, const float* beta_logit,
                               int bits, int64_t group, const float* dW_dq,
                               float* d_gamma_logit, float* d_beta_logit, float* d_s,
                               float* dW_tilde, void* ws, size_t ws_bytes, hipStream_t stream);
oq_status oq_lwc_fakequant_bwd_workspace_size(int64_t c_out, int64_t c_in, int64_t group,
                                              int want_d_s, size_t* bytes);

/* ---------------------------------------------------------------------------
 * Any weight quantiser (OQ_WQ_*), forward and straight-through backward, with
 * the arguments and outputs of oq_lwc_fakequant_fwd / _bwd (which are the
 * OQ_WQ_LWC case); p1, p2 and d_p1, d_p2 are the quantiser's two parameters
 * per group and their gradients.  Workspace of the backward:
 * oq_lwc_fakequant_bwd_workspace_size.
 */
oq_status oq_wquant_fakequant_fwd(int quantizer, const void* W, oq_dtype w_dt, int64_t c_out,
                                  int64_t c_in, const float* s, const float* p1, const float* p2,
                                  int bits, int64_t group, void* W_dq, oq_dtype dq_dt,
                                  uint8_t* codes, float* h, float* z, hipStream_t stream);
oq_status oq_wquant_fakequant_bwd(int quantizer, const void* W, oq_dtype w_dt, int64_t c_out,
                                  int64_t c_in, const float* s, const float* p1, const float* p2,
                                  int bits, int64_t group, const float* dW_dq, float* d_p1,
                                  float* d_p2, float* d_s, float* dW_tilde, void* ws,
                                  size_t ws_bytes, hipStream_t stream);
/* MinMax starting parameters of a quantiser per group of W~ = s (.) W:
 * PACT (hi, lo) = (max, min); LSQ (h, z) = Eq. 2's step and zero point at
 * clip strength 1; LWC logits 4.0 (Sec. 4.1 / the configurations' init).
 * p1, p2 [c_out, c_in/group] fp32 (outputs). */
oq_status oq_wquant_init(int quantizer, const void* W, oq_dtype w_dt, int64_t c_out, int64_t c_in,
                         const float* s, int bits, int64_t group, float* p1, float* p2,
                         hipStream_t stream);

/* ---------------------------------------------------------------------------
 * LET fold for a linear layer (Sec. 3.3, Eq. 3): W~ = s (.) W, B~ = B + delta W.
 *   W [c_out, c_in] (w_dt); B [c_out] fp32 | NULL; s, delta [c_in] fp32 | NULL
 *   W_tilde [c_out, c_in] (wt_dt) | NULL;  B_tilde [c_out] fp32 | NULL
 * B~ sums over input channels in fp64 and rounds once.
 */
oq_status oq_let_fold(const void* W, oq_dtype w_dt, const float* B, int64_t c_out, int64_t c_in,
                      const float* s, const float* delta, void* W_tilde, oq_dtype wt_dt,
                      float* B_tilde, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Per-token activation fake-quant with the LET input transform (Eq. 3-4;
 * Sec. 4.1: per-token asymmetric MinMax, i.e. Eq. 2 with gamma = beta = 1 on
 * each token row of X~ = (X - delta) / s, evaluated as (x - delta) * (1/s)).
 *   X      [T, C] (x_dt);  bits in [2,8], or 16 = no quantisation (X_dq = X~)
 *   X_dq   [T, C] (dq_dt) | NULL;  codes [T, C] uint8 | NULL;  h, z [T] fp32 | NULL
 */
oq_status oq_act_fakequant_fwd(const void* X, oq_dtype x_dt, int64_t T, int64_t C, int bits,
                               const float* s, const float* delta, void* X_dq, oq_dtype dq_dt,
                               uint8_t* codes, float* h, float* z, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Straight-through backward of oq_act_fakequant_fwd (Sec. 3.2, Eq. 2 at
 * gamma = beta = 1 per token row: only rint has derivative 1, the row's
 * max/min and the clamp are differentiated exactly; Eq. 3 for the LET input
 * transform X~ = (X - delta) / s, whose s and delta gradients are returned).
 *   dX_dq    [T, C] fp32          dL/dX^ (summed over every linear reading X^)
 *   dX_tilde [T, C] fp32 | NULL   dL/dX~
 *   d_s      [C] fp32 | NULL      input-path part of dL/ds    = -sum_t dL/dX~ * X~ / s
 *   d_delta  [C] fp32 | NULL      input-path part of dL/ddelta = -sum_t dL/dX~ / s
 * Workspace: oq_act_fakequant_bwd_workspace_size (0 bytes when d_s and d_delta are NULL).
 */
oq_status oq_act_fakequant_bwd(const void* X, oq_dtype x_dt, int64_t T, int64_t C, int bits,
                               const float* s, const float* delta, const float* dX_dq,
                               float* dX_tilde, float* d_s, float* d_delta,
                               void* ws, size_t ws_bytes, hipStream_t stream);
oq_status oq_act_fakequant_bwd_workspace_size(int64_t T, int64_t C, size_t* bytes);

/* ---------------------------------------------------------------------------
 * oq_act_fakequant_bwd without a workspace, for callers that cannot allocate
 * device memory (code under stream capture, serving loops, harnesses that
 * forbid hipMalloc).  Same arguments, outputs, kernels and results (bit for
 * bit) as oq_act_fakequant_bwd; the column partials of d_s / d_delta go to a
 * static device array of OQ_NOALLOC_SCRATCH_BYTES that the library holds on
 * each GPU it runs on until the process ends.  The call allocates nothing.
 *   Limit: when d_s or d_delta is wanted, the bytes that
 *   oq_act_fakequant_bwd_workspace_size reports for (T, C) must not exceed
 *   OQ_NOALLOC_SCRATCH_BYTES (else OQ_ERR_UNSUPPORTED, nothing launched);
 *   e.g. C = 4096 or 5120 at any T; C = 11008 only for T <= 381.
 *   Concurrency: every call on one GPU shares that GPU's array, so calls
 *   that overlap on one GPU (different streams or host threads) race; order
 *   them on one stream.  The array keeps the last call's partials; nothing
 *   in it needs to start at zero.
 */
#define OQ_NOALLOC_SCRATCH_BYTES (32u * 1024u * 1024u)
oq_status oq_act_fakequant_bwd_noalloc(const void* X, oq_dtype x_dt, int64_t T, int64_t C, int bits,
                                       const float* s, const float* delta, const float* dX_dq,
                                       float* dX_tilde, float* d_s, float* d_delta,
                                       hipStream_t stream);

/* ---------------------------------------------------------------------------
 * LET initialisation (Sec. 4.1: scale from SmoothQuant, shift from Outlier
 * Suppression+):  s_c = sqrt(max_t |X[t,c]|) / sqrt(max over the site's
 * linears and rows of |W[o,c]|), each max floored at 1e-5;  delta_c =
 * mean_t X[t,c] (fp64 sum).
 *   X [T, C] (x_dt); W_site: HOST array of n_site device pointers to
 *   [c_out_site[i], C] (w_dt) weights; s, delta [C] fp32 (outputs).
 */
oq_status oq_let_init(const void* X, oq_dtype x_dt, int64_t T, int64_t C,
                      const void* const* W_site, const int64_t* c_out_site, int n_site,
                      oq_dtype w_dt, float* s, float* delta, void* ws, size_t ws_bytes,
                      hipStream_t stream);
oq_status oq_let_init_workspace_size(int64_t T, int64_t C, const int64_t* c_out_site, int n_site,
                                     size_t* bytes);

/* ---------------------------------------------------------------------------
 * Full-precision target of one linear (Algorithm 1, the fp block output that
 * the quantised block is trained to match):  Y_T = W X^T + B, stored
 * channel-major [c_out, T] (the layout the calibration step consumes).
 *   X [T, c_in], W [c_out, c_in] (dt);  B [c_out] fp32 | NULL;  Y_T [c_out, T] (dt)
 * dt = OQ_BF16: bf16 matrix cores, fp32 accumulation, one bf16 rounding.
 */
oq_status oq_fp_target(const void* X, const void* W, oq_dtype dt, const float* B, int64_t T,
                       int64_t c_in, int64_t c_out, void* Y_T, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Plain matrix product C[M,N] = A[M,K] B[N,K]^T (both operands K-contiguous),
 * the building block of every linear in the step.  in_dt = OQ_BF16: matrix
 * cores with fp32 accumulation; OQ_F32: fp32 throughout.  C is out_dt.
 */
oq_status oq_matmul_nt(const void* A, const void* B, oq_dtype in_dt, int64_t M, int64_t N,
                       int64_t K, void* C, oq_dtype out_dt, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * The same product with either operand stored the other way round, read as
 * stored (the step's weight and input gradients use it on token-major X^ and
 * on W^ without transposing them):
 *   C[M,N] (fp32) = opA opB^T,  opA = A [M,K] (a_mn = 0) or A^T with A stored
 *   [K,M] (a_mn = 1);  opB = B [N,K] (b_mn = 0) or B^T with B stored [K,N].
 * bf16 only, dense row-major operands.  OQ_ERR_UNSUPPORTED when an operand
 * is MN-major and K is not a multiple of 64 or the MN side is not a multiple
 * of 8.
 */
oq_status oq_matmul(const void* A, int a_mn, const void* B, int b_mn, int64_t M, int64_t N,
                    int64_t K, float* C, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * AdamW update (Sec. 4.1: AdamW, zero weight decay; lr 5e-3 for the clipping
 * logits, 1e-2 for s and delta).  fp32, in place on p, m, v; step counts from 1.
 * Hyperparameters are doubles: the coefficients 1 - b1, 1 - b2 and the bias
 * corrections are formed in fp64 and rounded once to fp32.
 *   p = p*(1 - lr*wd);  m = b1*m + (1-b1)*g;  v = b2*v + (1-b2)*g*g
 *   p -= lr * (m / (1 - b1^step)) / (sqrt(v / (1 - b2^step)) + eps)
 */
oq_status oq_adamw_step(float* p, const float* g, float* m, float* v, int64_t n, double lr,
                        double beta1, double beta2, double eps, double wd, int step,
                        hipStream_t stream);

/* ---------------------------------------------------------------------------
 * One block-wise calibration step (Sec. 3.1 Eq. 1; Algorithm 1's inner loop
 * body: LET, LWC, forward of the quantised linears on x_q, squared error to
 * x_fp, straight-through backward, optional AdamW update).
 *
 * The block is its linear sub-graph: n_sites input tensors ("sites") and
 * n_linears linears; linear l reads site lin_site[l].  Linears of one site
 * must be consecutive.  LET (s, delta) applies per site; per-token
 * activation fake-quant applies to a site's input when site_act_bits < 16.
 * Loss = sum over linears of mean((Y_l - Y_fp,l)^2), Y_l = Q_a(X~) Q_w(W~)^T + B~.
 *
 * Ordering: the step is ordered on `stream` like a single launch.  At small
 * token counts (bf16, T <= 16384, every site's forward product within four
 * waves of 256 x 256 tiles, at most 4 sites) sites 1.. run on side streams
 * forked from `stream` with an event and joined back to it before the loss.
 * The side streams (non-blocking, default priority) and their events are
 * created on first use, once per device and host thread, and kept; each site
 * then has its own part of the workspace, so calls must not share one
 * workspace concurrently.
 */
#define OQ_MAX_SITES 8
#define OQ_MAX_LINEARS 16

typedef struct {
  int64_t tokens;                          /* T                                    */
  int n_sites, n_linears;
  oq_dtype dtype;                          /* OQ_BF16: bf16 X, W, Y_fp, bf16 MFMA;
                                              OQ_F32: fp32 everywhere             */
  int64_t site_width[OQ_MAX_SITES];        /* C of each site                       */
  int site_let[OQ_MAX_SITES];              /* 1 = LET on this site                 */
  int site_act_bits[OQ_MAX_SITES];         /* 2..8 (| OQ_ACT_SYM), or 16 = none     */
  int lin_site[OQ_MAX_LINEARS];
  int64_t lin_c_out[OQ_MAX_LINEARS];
  int lin_bits[OQ_MAX_LINEARS];
  int64_t lin_group[OQ_MAX_LINEARS];       /* group size along C_in (C_in = per channel) */
  int lin_quant[OQ_MAX_LINEARS];           /* weight quantiser: OQ_WQ_LWC (0, the default),
                                              OQ_WQ_PACT or OQ_WQ_LSQ; the params' and
                                              grads' gamma/beta slots then hold that
                                              quantiser's two parameters             */
} oq_block_desc;

typedef struct {                           /* device pointers                      */
  const void* W[OQ_MAX_LINEARS];           /* [c_out, C_site]                      */
  const float* B[OQ_MAX_LINEARS];          /* [c_out] | NULL                       */
  float* gamma_logit[OQ_MAX_LINEARS];      /* [c_out, C_site/group]                */
  float* beta_logit[OQ_MAX_LINEARS];
  float* s[OQ_MAX_SITES];                  /* [C_site], LET sites only             */
  float* delta[OQ_MAX_SITES];
} oq_block_params;

typedef struct {                           /* device pointers, outputs             */
  float* d_gamma_logit[OQ_MAX_LINEARS];    /* required                             */
  float* d_beta_logit[OQ_MAX_LINEARS];     /* required                             */
  float* d_s[OQ_MAX_SITES];                /* required on LET sites                */
  float* d_delta[OQ_MAX_SITES];            /* required on LET sites                */
  float* row_loss[OQ_MAX_LINEARS];         /* [c_out] | NULL: sum_t (Y - Y_fp)^2   */
} oq_block_grads;

typedef struct {                           /* AdamW state; NULL pointer = no update */
  float* m_gamma[OQ_MAX_LINEARS]; float* v_gamma[OQ_MAX_LINEARS];
  float* m_beta[OQ_MAX_LINEARS];  float* v_beta[OQ_MAX_LINEARS];
  float* m_s[OQ_MAX_SITES];       float* v_s[OQ_MAX_SITES];
  float* m_delta[OQ_MAX_SITES];   float* v_delta[OQ_MAX_SITES];
  int step;                                /* 1-based step number of this update   */
  double lr_lwc, lr_let, beta1, beta2, eps, wd;
  /* Iterative LWC/LET training (the ablation on training LWC and LET in
   * turn): OQ_FREEZE_LWC keeps the clipping logits fixed, OQ_FREEZE_LET keeps
   * s and delta fixed.  A frozen set is not updated and its AdamW m, v are
   * not touched; gradient work that only the frozen set needs is skipped
   * (a frozen LET skips the input-gradient path; a frozen LWC skips the
   * weight gradient of every site whose LET is absent or frozen), and the
   * frozen set's gradient outputs are then left unwritten.  0 = train both. */
  int frozen;
} oq_block_optim;
#define OQ_FREEZE_LWC 1
#define OQ_FREEZE_LET 2

oq_status oq_block_workspace_size(const oq_block_desc* desc, size_t* bytes);

/* The launch plan oq_block_calib_step takes for `desc` (a host query, nothing
 * launched), OQ_PLAN_FIELDS ints per site k at info[OQ_PLAN_FIELDS * k + i]:
 *   0  sites run concurrently on side streams      1  gradient products read
 *   X^ and dY^T as stored (no transposed copies)   2  K-split count of the
 *   weight gradient   3  K-split count of the forward product   4  LWC
 *   backward fused into the weight gradient's epilogue   5  input gradient
 *   reads a transposed copy of W^.   n_info >= OQ_PLAN_FIELDS * n_sites.  */
#define OQ_PLAN_FIELDS 6
oq_status oq_block_plan(const oq_block_desc* desc, int* info, int n_info);

/*   Y_fp_T : HOST array [n_linears] of device pointers, each [c_out, T] (Y_fp
 *            channel-major, as oq_fp_target writes it)
 *   X_q    : HOST array [n_sites] of device pointers, each [T, C_site]
 *   loss   : device float scalar (output)
 *   optim  : NULL = gradients only; else AdamW updates gamma/beta logits and s/delta in place
 */
oq_status oq_block_calib_step(const oq_block_desc* desc, const void* const* Y_fp_T,
                              const void* const* X_q, const oq_block_params* params,
                              const oq_block_grads* grads, const oq_block_optim* optim,
                              float* loss, void* ws, size_t ws_bytes, hipStream_t stream);

/* Algorithm 1's training loop for one block: `epochs` passes over
 * `n_segments` calibration segments in order (the paper's bs = 1 schedule is
 * 128 segments of 2048 tokens, 20 epochs), each one oq_block_calib_step with
 * the AdamW update.
 *   Y_fp_T : HOST array [n_segments * n_linears]; segment g's target of linear l
 *            at [g * n_linears + l], each [c_out, desc->tokens] channel-major
 *   X_q    : HOST array [n_segments * n_sites]; segment g's input of site k at
 *            [g * n_sites + k], each [desc->tokens, C_site]
 *   optim  : required; optim->step (>= 1) is the first step's count, the i-th
 *            step uses optim->step + i; the struct is not written
 *   losses : device float [epochs * n_segments]: the loss of every step, in order
 * Parameters, gradients, AdamW state and workspace as oq_block_calib_step (the
 * gradients hold the last step's).  Every pointer is validated before the first
 * launch; steps are issued in order on `stream`.
 */
oq_status oq_block_calibrate(const oq_block_desc* desc, int n_segments, int epochs,
                             const void* const* Y_fp_T, const void* const* X_q,
                             const oq_block_params* params, const oq_block_grads* grads,
                             const oq_block_optim* optim, float* losses, void* ws,
                             size_t ws_bytes, hipStream_t stream);

/* Checkpoint / resume of one block's calibration (Algorithm 1 trains each
 * block for many epochs; a run that stops can continue from its last saved
 * state).  The state is the learnable set Theta -- clipping logits per
 * linear, s and delta per LET site -- plus, with `opt`, the AdamW moments m,
 * v, the hyperparameters and the number of completed updates.
 *
 * oq_block_state_save copies the state to host memory and writes `path`
 * (first to path + ".tmp", then renamed over `path`, so an interrupted save
 * leaves the previous file intact).  File layout, little-endian: 8-byte
 * magic "OQCKPT\0\1"; int32 version (1), size of the shape record,
 * completed_steps, has-AdamW flag; the block's shape record (site widths,
 * LET flags, activation bits, linear sites, c_out, bits, groups,
 * quantisers); uint64
 * tensor count; with AdamW six doubles (lr_lwc, lr_let, beta1, beta2, eps,
 * wd); then per tensor uint32 kind, uint32 linear/site index, uint64
 * element count, uint64 FNV-1a hash of its bytes and the fp32 data.
 *
 * oq_block_state_load reads and verifies the whole file (magic, version,
 * shape equal to `desc`'s apart from the token count and dtype, every hash,
 * every size) before it writes any device buffer, then restores params (and
 * opt's m, v, hyperparameters, and opt->step = completed_steps + 1, the
 * number of the next update).  Both synchronise `stream`.  A failed load
 * changes nothing on the device.  Errors: OQ_ERR_INVALID_ARG (I/O, format,
 * mismatch), OQ_ERR_HIP.
 */
oq_status oq_block_state_save(const oq_block_desc* desc, const oq_block_params* params,
                              const oq_block_optim* opt, int completed_steps, const char* path,
                              hipStream_t stream);
oq_status oq_block_state_load(const oq_block_desc* desc, const oq_block_params* params,
                              oq_block_optim* opt, int* completed_steps, const char* path,
                              hipStream_t stream);

/* Algorithm 1's last step for one block ("obtain the quantised block"), on
 * its linear sub-graph: with the learned clipping logits and LET parameters,
 * each linear's weight is transformed (Eq. 3: s (.) W on LET sites) and
 * quantised by LWC (Eq. 2); its codes are written packed in the
 * oq_pack_codes layout with their h and z, ready for oq_packed_linear.
 *   packed  : HOST [n_linears] device pointers, each [c_out, C_site * bits / 8] u8
 *   h, z    : HOST [n_linears] device pointers, each [c_out, C_site / group] fp32
 *   B_tilde : HOST [n_linears] device pointers [c_out] fp32, or NULL (array or
 *             entry): the folded bias B + delta W on LET sites, else B (0 without B)
 * The deployed linear then reads X~ = (X - delta) / s on LET sites (Eq. 3).
 * C_site % 32 == 0 (else OQ_ERR_INVALID_ARG); every linear's bits <= 7 and
 * group % 32 == 0, what oq_packed_linear accepts (else OQ_ERR_UNSUPPORTED).
 * Workspace: oq_block_export_workspace_size bytes, 16-byte aligned (the
 * largest linear's u8 codes).  Other errors as oq_block_calib_step.
 */
oq_status oq_block_export_workspace_size(const oq_block_desc* desc, size_t* bytes);
oq_status oq_block_export(const oq_block_desc* desc, const oq_block_params* params,
                          uint8_t* const* packed, float* const* h, float* const* z,
                          float* const* B_tilde, void* ws, size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * LET absorbed into the operation that produces a site's input (Sec. 3.3:
 * after calibration s and delta fold into the preceding normalisation or
 * linear layer, so the deployed block runs no extra transform; on the
 * [v, o] pair the attention probabilities sum to 1 over keys, so a shift of
 * V passes through them).  Row c of P [C, n] in p_dt (a normalisation's
 * gain is n = 1; a previous linear's weight [C, c_in_prev] has the site's
 * channels as its output rows) becomes P[c, :] * (1/s[c]), and its bias
 * b [C] fp32 | NULL (0) becomes (b[c] - delta[c]) * (1/s[c]) in b_out [C]
 * fp32 -- the same fp32 order as the activation transform (x - delta)*(1/s),
 * so the absorbed producer emits X~ = (X - delta)/s.  s, delta [C] fp32 |
 * NULL (ones / zeros).  P_out may be NULL (bias only); P_out may equal P.
 */
oq_status oq_let_absorb(const void* P, oq_dtype p_dt, const float* b, int64_t C, int64_t n,
                        const float* s, const float* delta, void* P_out, float* b_out,
                        hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Deployment of the calibrated weights (Sec. 4.5 and Table "tab:speed":
 * weight-only WxA16 models whose weights are stored as Eq.2's integer codes
 * W_q with one step size h and zero point z per group).
 *
 * oq_pack_codes: codes [c_out, c_in] u8 -> packed [c_out, c_in * bits / 8] u8,
 * both device memory owned by the caller.  Row o's codes form one
 * little-endian bit string: code j occupies bits j*bits .. j*bits + bits - 1,
 * and bit k of the string is bit (k mod 8) of byte k / 8; rows follow each
 * other.  Only the low `bits` bits of each code are stored.
 * Supported: bits 2..8 (else OQ_ERR_UNSUPPORTED); c_in % 32 == 0; both
 * pointers 16-byte aligned (else OQ_ERR_INVALID_ARG).  c_out == 0 is a no-op
 * that accepts NULL pointers.
 */
oq_status oq_pack_codes(const uint8_t* codes, int64_t c_out, int64_t c_in, int bits,
                        uint8_t* packed, hipStream_t stream);

/* oq_packed_linear: Y = X W^T + B with W[o, c] = (q[o, c] - z[o, g]) * h[o, g],
 * g = c / group, the dequantisation of Eq.2, q read from `packed`.
 *   X      : bf16 [n_tok, c_in] (x_dt must be OQ_BF16, else OQ_ERR_UNSUPPORTED)
 *   packed : u8 [c_out, c_in * bits / 8] in the oq_pack_codes layout
 *   h, z   : fp32 [c_out, c_in / group], as oq_lwc_fakequant_fwd writes them
 *   B      : fp32 [c_out] | NULL
 *   Y      : [n_tok, c_out] in y_dt (fp32 or bf16), overwritten
 * Supported: bits 2..7 and c_in <= 65536 (else OQ_ERR_UNSUPPORTED); c_in % 32
 * == 0; group % 32 == 0 dividing c_in; every pointer 16-byte aligned (else
 * OQ_ERR_INVALID_ARG).  Any n_tok >= 0: below 8 tokens (or for groups other
 * than 128) the vector kernel, sized for decoding, one launch per 8 tokens;
 * from 8 tokens with groups of 128 the matrix-core kernel, one launch per 32
 * tokens (16 past 32768 input channels); each launch reads the packed weights
 * once.  n_tok == 0 or c_out == 0
 * is a no-op that accepts NULL pointers.  Products of codes and activations
 * are exact in fp32 and the sums run in a fixed order, so results are
 * reproducible (on matrix cores a token's outputs do not depend on the other
 * tokens of its batch).
 */
oq_status oq_packed_linear(const void* X, oq_dtype x_dt, int64_t n_tok, int64_t c_in,
                           const uint8_t* packed, int bits, int64_t group, const float* h,
                           const float* z, const float* B, int64_t c_out, void* Y,
                           oq_dtype y_dt, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Causal multi-head attention of the block (Sec. 3.3, Eq. 5: the attention
 * operation on the quantised Q^, K^, V^), on bf16 matrix cores.
 *   Q [T, H d], K, V [T, Hkv d] bf16 device, token-major, heads side by side;
 *   T = n_seq * S tokens, sample after sample; query head h reads key/value
 *   head h / (H / Hkv).  O [T, H d] fp32 = softmax(Q K^T / sqrt(d) + causal
 *   mask) V per sample and head.  LSE [H, T] fp32: per query the log-sum-exp
 *   of its logits in base 2 of t = q.k log2(e)/sqrt(d) (kept for the backward).
 * softmax_bits = 16: the probabilities enter the product with V as bf16
 * weights 2^(t - ceil(max t)) and O is divided by the sum of those rounded
 * weights (an exact weighted mean of V rows); pstat may be NULL.
 * softmax_bits in 2..8 (the ablation on quantising the softmax output,
 * Table tab:ablation_softmax): each query row of probabilities P = 2^(t - LSE),
 * its S entries with the causally masked zeros, goes through the activation
 * quantiser (per-row asymmetric MinMax, Eq. 2 with gamma = beta = 1) and the
 * dequantised row multiplies V as bf16 operands, not renormalised.  pstat
 * [H, T, 4] fp32 (16-byte aligned) receives per row (max P, min P, and the
 * lowest key index holding each, as int32 bit patterns) for the backward.
 * Backward: dO [T, H d] bf16 -> dQ [T, H d], dK, dV [T, Hkv d] fp32 (dK and dV
 * summed over the query heads of each group), from the probabilities
 * recomputed with LSE; D = sum_j P_ij dP_ij is formed from those same
 * probabilities; P (or its quantised row) enters the dV product as bf16, dS
 * the dQ and dK products as a pair of bf16 terms (hi + lo); with a quantised
 * softmax dP passes the quantiser's straight-through backward first (the
 * row's max / min gradients to the keys in pstat).  Deterministic (no
 * atomics).  Workspace: [H, T] fp32 (D), three times that with a quantised
 * softmax.
 * Supported: d in {64, 128}, S a multiple of 64, T a multiple of S.
 */
oq_status oq_attention_fwd(const void* Q, const void* K, const void* V, int64_t T, int64_t S,
                           int H, int Hkv, int head_dim, int softmax_bits, float* O, float* LSE,
                           float* pstat, hipStream_t stream);
oq_status oq_attention_bwd_workspace_size(int64_t T, int H, int softmax_bits, size_t* bytes);
oq_status oq_attention_bwd(const void* Q, const void* K, const void* V, const void* dO,
                           const float* LSE, const float* pstat, int64_t T, int64_t S, int H,
                           int Hkv, int head_dim, int softmax_bits, float* dQ, float* dK, float* dV,
                           void* ws, size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * One calibration step over a whole LLaMA transformer block (Eq. 1 with F
 * the block itself; Algorithm 1's inner-loop body):
 *   x1 = RMSNorm(h0) g1;  q, k, v = Q_w(W~) Q_a((x1 - delta1)/s1) + B~
 *   q, k <- RoPE (pairs (i, i + d/2) of each head, position = token mod S)
 *   Q~ = q / s_a, K~ = k * s_a (Eq. 5, after RoPE; s_a per key-head channel,
 *   shared by the query heads of its group); Q^, K^, V^ = Q_a(Q~, K~, v)
 *   o = causal softmax(Q^ K^T / sqrt(d)) V^ per sample and head
 *   h1 = h0 + Q_w(W_o~) Q_a((o - delta2)/s2) + B~_o
 *   x3 = RMSNorm(h1) g2; x4 = SiLU(gate) * up with gate, up from site 3
 *   h2 = h1 + Q_w(W_d) Q_a(x4);  loss = mean over T x D of (h2 - target)^2
 * with the straight-through backward to every clipping logit, s, delta and
 * s_a, and an optional AdamW update.  Activations bf16 at every matrix-core
 * operand, fp32 residual stream and accumulation.
 *   h0, target : bf16 [T, D] device (the block's quantised-model input X_q and
 *                its full-precision output X_fp, Algorithm 1)
 * Supported: head_dim D/H in {64, 128}; S a multiple of 64; T a multiple of
 * S; H a multiple of Hkv; every linear's c_in a multiple of 64; bits 2..8,
 * groups as oq_lwc_fakequant_fwd.  Workspace: oq_llama_workspace_size.
 * The step's backward runs each site's weight side (weight gradient, LWC
 * backward, LET weight and bias paths) on a side stream (non-blocking,
 * default priority, created once per device and host thread) forked from
 * `stream` and joined back to it before the step returns, so the step
 * orders on `stream` like one launch.
 */
#define OQ_LLAMA_LINEARS 7   /* q, k, v, o, gate, up, down */
typedef struct {
  int64_t tokens, seq_len;            /* T = n_seq * seq_len                       */
  int64_t hidden, ffn;                /* D, F                                      */
  int heads, kv_heads;                /* H, Hkv                                    */
  float norm_eps, rope_base;          /* RMSNorm epsilon, RoPE base (10000)        */
  int w_bits[OQ_LLAMA_LINEARS];
  int64_t w_group[OQ_LLAMA_LINEARS];  /* group along c_in (c_in = per channel)     */
  int act_bits;                       /* 2..8 (| OQ_ACT_SYM): Q_a on the four linear
                                         inputs and on Q~, K~, V; 16 = none       */
  int let;                            /* 1: LET on the q/k/v, o, gate/up inputs and s_a */
  int softmax_bits;                   /* 2..8: Q_a on each query row of the softmax
                                         output (as oq_attention_fwd); 16 = none */
} oq_llama_desc;

typedef struct {                      /* device pointers                            */
  const void* W[OQ_LLAMA_LINEARS];    /* bf16 [c_out, c_in]                         */
  const float* norm1;                 /* RMSNorm gains [D] fp32 (frozen)            */
  const float* norm2;
  float* gamma_logit[OQ_LLAMA_LINEARS]; /* [c_out, c_in / group]                    */
  float* beta_logit[OQ_LLAMA_LINEARS];
  float* s[3];                        /* [D], [H d], [D]  (LET only)                */
  float* delta[3];
  float* s_a;                         /* [Hkv d]           (LET only)               */
} oq_llama_params;

typedef struct {                      /* device outputs                              */
  float* d_gamma_logit[OQ_LLAMA_LINEARS];
  float* d_beta_logit[OQ_LLAMA_LINEARS];
  float* d_s[3];
  float* d_delta[3];
  float* d_s_a;
} oq_llama_grads;

typedef struct {                      /* AdamW state, as oq_block_optim             */
  float* m_gamma[OQ_LLAMA_LINEARS]; float* v_gamma[OQ_LLAMA_LINEARS];
  float* m_beta[OQ_LLAMA_LINEARS];  float* v_beta[OQ_LLAMA_LINEARS];
  float* m_s[3]; float* v_s[3]; float* m_delta[3]; float* v_delta[3];
  float* m_s_a; float* v_s_a;
  int step;
  double lr_lwc, lr_let, beta1, beta2, eps, wd;
} oq_llama_optim;

oq_status oq_llama_workspace_size(const oq_llama_desc* desc, size_t* bytes);
oq_status oq_llama_block_step(const oq_llama_desc* desc, const void* h0, const void* target,
                              const oq_llama_params* params, const oq_llama_grads* grads,
                              const oq_llama_optim* optim, float* loss, void* ws,
                              size_t ws_bytes, hipStream_t stream);

/* Algorithm 1's training loop for one block: `epochs` passes over the
 * samples in order, one oq_llama_block_step with the AdamW update per sample
 * (batch size 1, Sec. 4.1).  h0[j], target[j]: sample j's block input X_q and
 * its full-precision block output, bf16 [tokens, hidden] device, 16-byte
 * aligned, each desc->tokens tokens.  The AdamW steps count from optim->step
 * (>= 1) on; losses: device fp32 [epochs * n_samples], step i = epoch *
 * n_samples + j.  Parameters are updated in place; grads hold the last step's
 * gradients.  Pointers are checked before the first launch; a failing step
 * returns its status with the earlier steps applied.  Same workspace as the
 * step. */
oq_status oq_llama_calibrate(const oq_llama_desc* desc, int n_samples, int epochs,
                             const void* const* h0, const void* const* target,
                             const oq_llama_params* params, const oq_llama_grads* grads,
                             const oq_llama_optim* optim, float* losses, void* ws,
                             size_t ws_bytes, hipStream_t stream);

/* The block's forward alone, for Algorithm 1's propagation from block to
 * block: quantised = 0 gives the full-precision block (W as given, no LET,
 * no quantiser: X_fp <- B(X_fp)); quantised = 1 the quantised block with the
 * learned parameters (X_q <- B_q(X_q)).  h_out: bf16 [T, D], may not alias
 * h0.  Same workspace as the step. */
oq_status oq_llama_block_forward(const oq_llama_desc* desc, const void* h0,
                                 const oq_llama_params* params, int quantised, void* h_out,
                                 void* ws, size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Kernel timing on the launching stream (HIP events around each launch).
 * Kinds: 0 forward GEMM, 1 weight-gradient GEMM, 2 input-gradient GEMM,
 * 3 LWC forward, 4 LWC backward, 5 activation quant forward, 6 activation
 * quant backward, 7 transposes, 8 other, 9 the packed linear, 10 attention
 * forward, 11 attention backward.  oq_profile_read synchronises the
 * recorded events and returns launch count, total milliseconds and the
 * algorithmic work (FLOP for GEMMs, bytes for the others) of that kind.
 */
#define OQ_PROF_KINDS 12
oq_status oq_profile_enable(int on);
oq_status oq_profile_reset(void);
oq_status oq_profile_read(int kind, int64_t* launches, double* total_ms, double* work);

#ifdef __cplusplus
}
#endif
#endif /* OQ_H */
