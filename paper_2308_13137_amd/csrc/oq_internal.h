// Host-side launchers shared between the kernel files and the C ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

namespace oq {

enum ProfKind {
  PK_GEMM_FWD = 0, PK_GEMM_WGRAD = 1, PK_GEMM_DGRAD = 2, PK_LWC_FWD = 3, PK_LWC_BWD = 4,
  PK_ACT_FWD = 5, PK_ACT_BWD = 6, PK_TRANSPOSE = 7, PK_OTHER = 8,
  PK_ATTN_FWD = 10, PK_ATTN_BWD = 11
};

// Kernel timing: when enabled, brackets a launch with events on its stream.
struct ProfScope {
  ProfScope(int kind, hipStream_t s, double work);
  ~ProfScope();
  int kind;
  hipStream_t stream;
  double work;
  hipEvent_t e0, e1;
  bool on;
};

// ---------------------------------------------------------------- GEMM: C = A B^T
// The forward epilogue of the calibration step: per output row m (an output
// channel of one of up to MAX_SEG linears stacked along M) and column n (a token)
//   y = acc + bias[m];  r = y - yfp[m][n];  dy = bf16(r * scale);  store dy
// and per (row, column tile) the partial sums of r^2 and of dy.
constexpr int MAX_SEG = 4;
struct ResidArgs {
  int nseg;
  int64_t seg_end[MAX_SEG];        // exclusive row end of each linear
  const void* yfp[MAX_SEG];        // [rows_l, ld_yfp], channel-major target
  float scale[MAX_SEG];            // 2 / (T * c_out_l)
  int64_t seg_begin[MAX_SEG];
  int64_t ld_yfp;
  const float* bias;               // [M] | nullptr
  void* dy;                        // [M, ld_dy]
  int64_t ld_dy;
  float* part_sq;                  // [M, ntn]
  float* part_dy;                  // [M, ntn] | nullptr
  int ntn;                         // column tiles (set by the launcher)
};

// Column-tile width of the row partials written by the forward epilogue.
int gemm_part_tile_n(bool bf16);

hipError_t gemm_nt_f32out(const void* A, const void* B, bool bf16, int64_t M, int64_t N, int64_t K,
                          int64_t lda, int64_t ldb, float* C, int64_t ldc, hipStream_t st);
// bf16 C[M,N] = op(A) op(B)^T into fp32 with either operand stored MN-major
// (a_mn: A as [K, M] with row stride lda; b_mn: B as [K, N] with row stride
// ldb), read straight from that layout.  gemm_mn_supported tells whether the
// shapes qualify (K a multiple of 64 and aligned strides).  With splits > 1
// the K range is cut into that many equal parts (each a multiple of 64) and
// part s writes its own partial product at C + s * split_stride; the caller
// sums the parts (sum_partials).
bool gemm_mn_supported(bool a_mn, bool b_mn, int64_t M, int64_t N, int64_t K, int64_t lda,
                       int64_t ldb);
// K-split count (1, 2, 4 or 8) for gemm_f32out_mn on an M x N output: the one
// whose whole waves of 256 x 256 tiles over 256 compute units, plus the
// partial-sum pass, take the least modelled time.
int gemm_mn_splits(bool a_mn, bool b_mn, int64_t M, int64_t N, int64_t K, int64_t lda,
                   int64_t ldb);
hipError_t gemm_f32out_mn(const void* A, bool a_mn, const void* B, bool b_mn, int64_t M,
                          int64_t N, int64_t K, int64_t lda, int64_t ldb, float* C, int64_t ldc,
                          hipStream_t st, int splits = 1, int64_t split_stride = 0);
hipError_t gemm_nt_store(const void* A, const void* B, bool bf16, int64_t M, int64_t N, int64_t K,
                         int64_t lda, int64_t ldb, void* C, bool c_bf16, int64_t ldc,
                         const float* bias, hipStream_t st);
hipError_t gemm_nt_resid(const void* A, const void* B, bool bf16, int64_t M, int64_t N, int64_t K,
                         int64_t lda, int64_t ldb, ResidArgs ra, hipStream_t st);
// The same forward split over K (bf16): `splits` fp32 partial products go to
// parts [splits, M, N], then one pass sums them in order and applies the
// residual epilogue.  gemm_resid_splits picks the count (1 = do not split)
// for 256 compute units: few output tiles and a long K.
int gemm_resid_splits(int64_t M, int64_t N, int64_t K);
hipError_t gemm_nt_resid_split(const void* A, const void* B, int64_t M, int64_t N, int64_t K,
                               int64_t lda, int64_t ldb, ResidArgs ra, float* parts, int splits,
                               hipStream_t st);

// The weight gradient with the LWC straight-through backward in its epilogue
// (no LET, power-of-two groups of 8..256 weights).  The product dW^ = dY^T X^
// over rows m of up to MAX_SEG linears stacked along M is never stored: per
// (row, group) the epilogue forms S_h = sum g ((q - z) - m u) and
// S_z = sum g (1 - m) from the accumulators, the bf16 weights and the group
// statistics the forward wrote, and writes the logit gradients.
struct LwcArgs {
  int nseg;
  int64_t seg_begin[MAX_SEG], seg_end[MAX_SEG];
  const uint16_t* W[MAX_SEG];      // bf16 [rows_l, C]
  float* dgl[MAX_SEG];             // [rows_l, ng] outputs
  float* dbl[MAX_SEG];
  const float4* gstat;             // [M, ng] pairs {max, min, h, z}, {gamma, beta, 1/h, 0}
  int64_t C;
  int group, ng;
  float qmax;
};
bool gemm_wgrad_lwc_supported(int64_t M, int64_t C, int64_t K, int group);
// dY^T [M, K] K-contiguous (lda), X^ [K, C] read C-contiguous (ldb).
hipError_t gemm_wgrad_lwc(const void* dyT, const void* x, int64_t M, int64_t C, int64_t K,
                          int64_t lda, int64_t ldb, const LwcArgs& la, hipStream_t st);

// ---------------------------------------------------------------- quantisers
// LWC forward on rows [0, c_out) of one weight.  Returns hipErrorInvalidValue
// when (c_in, group) is outside the supported set.
// gstat (power-of-two groups without s only) receives two float4 per group:
// {max, min, h, z} and {gamma, beta, 1/h, 0}.
// quant: WQ_LWC (gl, bl = clip-strength logits), WQ_PACT (gl, bl = upper and
// lower thresholds), WQ_LSQ (gl, bl = step and zero point); see common.h.
hipError_t lwc_fwd(const void* W, bool w_bf16, int64_t c_out, int64_t c_in, const float* s,
                   const float* gl, const float* bl, int bits, int64_t group, void* W_dq,
                   bool dq_bf16, uint8_t* codes, float* h, float* z, hipStream_t st,
                   float4* gstat = nullptr, int quant = 0);
// LWC backward.  When ds_parts != nullptr each block writes one partial row
// [c_in] of sum_o dW~[o,c]*W[o,c] into ds_parts; the number of rows written is
// lwc_bwd_nparts(c_out).
int64_t lwc_bwd_nparts(int64_t c_out);
// With parts > 1 (only where lwc_bwd_sums_parts holds) dW holds `parts`
// partial products spaced part_stride floats apart, summed in order on load.
bool lwc_bwd_sums_parts(int64_t c_out, int64_t c_in, int64_t group, bool has_s, bool want_ds);
hipError_t lwc_bwd(const void* W, bool w_bf16, int64_t c_out, int64_t c_in, const float* s,
                   const float* gl, const float* bl, int bits, int64_t group, const float* dW,
                   float* dgl, float* dbl, float* dW_tilde, float* ds_parts, hipStream_t st,
                   int parts = 1, int64_t part_stride = 0, int quant = 0);
bool quant_shape_supported(int64_t c_in, int64_t group);
// MinMax starting parameters of a weight quantiser variant, per group.
hipError_t wquant_init(const void* W, bool w_bf16, int64_t c_out, int64_t c_in, const float* s,
                       int bits, int64_t group, int quant, float* p1, float* p2, hipStream_t st);

// Activation fake-quant (per token row), LET transform included.
// sym: symmetric absmax quantiser (zero point 2^(bits-1)) in place of MinMax.
hipError_t act_fwd(const void* X, bool x_bf16, int64_t T, int64_t C, int bits, const float* s,
                   const float* delta, void* X_dq, bool dq_bf16, uint8_t* codes, float* h,
                   float* z, hipStream_t st, bool sym = false);
int64_t act_bwd_nparts(int64_t T);
hipError_t act_bwd(const void* X, bool x_bf16, int64_t T, int64_t C, int bits, const float* s,
                   const float* delta, const float* dXdq, float* dXt, float* p_sx, float* p_s1,
                   hipStream_t st, bool sym = false);

// ---------------------------------------------------------------- elementwise / reductions
hipError_t transpose(const void* in, int64_t rows, int64_t cols, int64_t ld_in, void* out,
                     int64_t ld_out, int elem_bytes, hipStream_t st);
hipError_t let_fold(const void* W, bool w_bf16, const float* B, int64_t c_out, int64_t c_in,
                    const float* s, const float* delta, void* Wt, bool wt_bf16, float* Bt,
                    hipStream_t st);
// LET absorbed into the producer of a site's input: Pout[c,:] = P[c,:]*(1/s[c]),
// bout[c] = (b[c] - delta[c])*(1/s[c]); P is [C, n] (n = 1 for a norm gain).
hipError_t let_absorb(const void* P, bool p_bf16, const float* b, int64_t C, int64_t n,
                      const float* s, const float* delta, void* Pout, float* bout,
                      hipStream_t st);
// out_parts[b][c] = sum over rows o of block b of wt[o] * W[o,c]
int64_t wcolsum_nparts(int64_t rows);
hipError_t wcolsum(const void* W, bool w_bf16, int64_t rows, int64_t cols, const float* wt,
                   float* out_parts, hipStream_t st);
// LET gradient finish, per column c (fp64, fixed order):
//   d_s[c]     = sum_b pw[b][c] - (sum_b psx[b][c]) / s[c]
//   d_delta[c] = sum_b pb[b][c] - (sum_b ps1[b][c]) / s[c]
hipError_t let_grad_finish(int64_t C, const float* s, const float* pw, int64_t npw,
                           const float* psx, const float* ps1, int64_t npa, const float* pb,
                           int64_t npb, float* d_s, float* d_delta, hipStream_t st);
// Row sums of the forward partials: rl[m] = sum_j psq[m][j] (fp64), and
// dbt[m] = sum_j pdy[m][j] when pdy != nullptr.
hipError_t row_partials(const float* psq, const float* pdy, int64_t M, int ntn, double* rl,
                        float* dbt, hipStream_t st);
// loss = sum over linears l of sum_{m in l} rl[m] / n_l;  row_loss outputs optional.
struct LossArgs {
  int nlin;
  int64_t row_begin[16], row_end[16];
  double inv_n[16];
  float* row_loss[16];
};
hipError_t loss_finish(const double* rl, LossArgs la, float* loss, hipStream_t st);
// AdamW with its fp32 coefficients formed in fp64 on the host.
struct AdamCoef {
  float lr, b1, omb1, b2, omb2, eps, decay, bc1, bc2;
};
AdamCoef adam_coef(double lr, double b1, double b2, double eps, double wd, int step);
// Up to ADAM_MAX tensors updated by one launch; set[k] picks coefficient set
// 0 or 1; block_begin is filled in by adamw_multi.
constexpr int ADAM_MAX = 48;
struct AdamList {
  int n;
  float* p[ADAM_MAX];
  const float* g[ADAM_MAX];
  float* m[ADAM_MAX];
  float* v[ADAM_MAX];
  int64_t len[ADAM_MAX];
  int set[ADAM_MAX];
  int block_begin[ADAM_MAX];
};
hipError_t adamw_multi(const AdamList& L, AdamCoef c0, AdamCoef c1, hipStream_t st);
// In place over the first of `parts` fp32 partials spaced `stride` apart:
// c[i] = ((c[i] + c[i + stride]) + ...) in that order, i < n.
hipError_t sum_partials(float* c, int64_t n, int parts, int64_t stride, hipStream_t st);
// d = the sum of the parts c, c + stride, ... (fixed order); d may be c.
hipError_t sum_partials_to(const float* c, float* d, int64_t n, int parts, int64_t stride,
                           hipStream_t st);
hipError_t adamw(float* p, const float* g, float* m, float* v, int64_t n, AdamCoef c,
                 hipStream_t st);
// LET initialisation pieces
int64_t colstat_nparts(int64_t rows);
hipError_t colstat(const void* X, bool bf16, int64_t rows, int64_t cols, float* amax_parts,
                   double* sum_parts, hipStream_t st);
hipError_t let_init_finish(int64_t C, int64_t T, const float* ax_parts, int64_t nax,
                           const double* sum_parts, const float* aw_parts, int64_t naw, float* s,
                           float* delta, hipStream_t st);

// ---------------------------------------------------------------- whole-block pieces
// Causal attention (bf16 matrix cores), head_dim 64 or 128, S a multiple of 64.
bool attn_supported(int64_t T, int S, int H, int Hkv, int dh);
// p_bits < 16: each query row of probabilities goes through Q_a before the
// product with V; pstat [H, T] float4 = (max P, min P, their lowest indices as
// int bits) is written by the forward and read by the backward.
hipError_t attn_fwd(const void* Q, const void* K, const void* V, int64_t T, int S, int H, int Hkv,
                    int dh, int p_bits, float* O, float* LSE, float* pstat, hipStream_t st);
// ws: attn_bwd_ws_floats fp32 scratch (D = sum_j P_ij dP_ij per query row, and
// with p_bits < 16 the row's max / min gradients); dQ [T, H dh], dK, dV
// [T, Hkv dh] fp32 outputs.
size_t attn_bwd_ws_floats(int64_t T, int H, int p_bits);
hipError_t attn_bwd(const void* Q, const void* K, const void* V, const void* dO, const float* LSE,
                    const float* pstat, int64_t T, int S, int H, int Hkv, int dh, int p_bits,
                    float* ws, float* dQ, float* dK, float* dV, hipStream_t st);
hipError_t rmsnorm_fwd(const void* h, bool h_bf16, const float* g, int64_t T, int64_t D, float eps,
                       float* x, float* rstd, hipStream_t st);
hipError_t rmsnorm_bwd(const void* h, bool h_bf16, const float* g, const float* rstd,
                       const float* dxt, const float* s, const float* dres, int64_t T, int64_t D,
                       float* dh, hipStream_t st);
// RoPE angle table of one sample: tab [S, dh/2] float2 (cos, sin).
hipError_t rope_table(int S, int dh, float base, float* tab, hipStream_t st);
hipError_t qkv_post(const float* qkv, const float* b, int64_t T, int S, int H, int Hkv, int dh,
                    const float* tab, const float* sa, float* Qt, float* Kt, float* V,
                    hipStream_t st);
hipError_t qkv_post_bwd(const float* dQt, const float* dKt, const float* dV, int64_t T, int S,
                        int H, int Hkv, int dh, const float* tab, const float* sa, void* dqkv,
                        hipStream_t st);
hipError_t sa_grad_finish(const float* pq, int64_t nq, const float* pk, int64_t nk, int H, int Hkv,
                          int dh, const float* sa, float* dsa, hipStream_t st);
hipError_t silu_mul(float* gu, const float* b, int64_t T, int64_t F, float* x4, hipStream_t st);
hipError_t silu_mul_bwd(const float* gu, const float* dx4, int64_t T, int64_t F, void* dgu,
                        hipStream_t st);
hipError_t resid_add(const void* base, bool base_bf16, const float* y, const float* b, int64_t T,
                     int64_t D, float* out, hipStream_t st);
hipError_t block_loss(const float* h2, const void* tgt, int64_t T, int64_t D, float* dh,
                      void* dh16, double* rows, float* loss, hipStream_t st);
hipError_t scale_to_bf16(const float* in, const float* s, int64_t T, int64_t C, void* out,
                         hipStream_t st);
hipError_t colsum_finish(const double* parts, int64_t n, int64_t C, float* out, hipStream_t st);

}  // namespace oq
