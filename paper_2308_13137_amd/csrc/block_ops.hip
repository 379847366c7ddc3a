// The non-linear pieces of a whole LLaMA block for the calibration step:
// RMSNorm (forward, backward), the q/k/v epilogue (bias, RoPE, the [Q, K]
// scale of Eq. 5) and its backward, SiLU gating, residual adds, the loss on
// the block output, and fp32 -> bf16 operand conversions.  All elementwise or
// row-wise, HBM-bound; every reduction has a fixed order (no atomics).
#include <math.h>

#include "common.h"
#include "oq_internal.h"

namespace oq {
namespace {

constexpr int BT = 256;

OQ_DEV float block_sum(float v, float* sh) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  return ((sh[0] + sh[1]) + sh[2]) + sh[3];
}

// ------------------------------------------------------------------ RMSNorm
// One workgroup per token row: x = h * rstd * g, rstd = 1/sqrt(mean(h^2) + eps).
// h is fp32 (the residual stream) or bf16 (the block's input).
template <typename TH>
__global__ __launch_bounds__(BT) void rmsnorm_fwd_kernel(const TH* __restrict__ h,
                                                         const float* __restrict__ g, int64_t D,
                                                         float eps, float* __restrict__ x,
                                                         float* __restrict__ rstd) {
  __shared__ float sh[4];
  const int64_t row = blockIdx.x;
  const TH* hr = h + row * D;
  float s = 0.f;
  for (int64_t c = threadIdx.x; c < D; c += BT) {
    const float v = load1(hr + c);
    s += v * v;
  }
  s = block_sum(s, sh);
  const float r = float(1.0 / sqrt(double(s) / double(D) + double(eps)));
  for (int64_t c = threadIdx.x; c < D; c += BT) x[row * D + c] = load1(hr + c) * r * g[c];
  if (threadIdx.x == 0) rstd[row] = r;
}

// dh = dres + rstd (g dx) - h rstd^3 sum(g dx h) / D, with dx = dxt / s when a
// LET scale is given (X~ = (X - delta)/s upstream of the linears).
template <typename TH>
__global__ __launch_bounds__(BT) void rmsnorm_bwd_kernel(const TH* __restrict__ h,
                                                         const float* __restrict__ g,
                                                         const float* __restrict__ rstd,
                                                         const float* __restrict__ dxt,
                                                         const float* __restrict__ s,
                                                         const float* __restrict__ dres, int64_t D,
                                                         float* __restrict__ dh) {
  __shared__ float sh[4];
  const int64_t row = blockIdx.x;
  const float r = rstd[row];
  float dot = 0.f;
  for (int64_t c = threadIdx.x; c < D; c += BT) {
    const float dx = s ? dxt[row * D + c] / s[c] : dxt[row * D + c];
    dot += g[c] * dx * load1(h + row * D + c);
  }
  dot = block_sum(dot, sh);
  const float k = r * r * r * dot / float(D);
  for (int64_t c = threadIdx.x; c < D; c += BT) {
    const float dx = s ? dxt[row * D + c] / s[c] : dxt[row * D + c];
    const float v = r * (g[c] * dx) - load1(h + row * D + c) * k;
    dh[row * D + c] = (dres ? dres[row * D + c] : 0.0f) + v;
  }
}

// ------------------------------------------------------------------ q/k/v epilogue
// QKV [T, (H + 2 Hkv) d] fp32 from the stacked product (q | k | v), bias b
// (B~ of the LET fold) or null.  Q~ = RoPE(q + b) / s_a (s_a of the query
// head's key group), K~ = RoPE(k + b) * s_a, V = v + b.  RoPE turns the pair
// (i, i + d/2) of each head by pos * base^(-2i/d), pos = token mod S.
// One thread per (token, pair) of q and k heads and per v element pair.
// RoPE angles of one sample: tab[pos * (d/2) + p] = (cos, sin) of
// pos * base^(-2p/d), evaluated in fp64 and rounded to fp32 (computed once per
// step; the rotation kernels read it from L2).
__global__ __launch_bounds__(BT) void rope_table_kernel(int S, int dh, float base,
                                                        float2* __restrict__ tab) {
  const int half = dh / 2;
  const int64_t i = int64_t(blockIdx.x) * BT + threadIdx.x;
  if (i >= int64_t(S) * half) return;
  const int pos = int(i / half), p = int(i % half);
  const double ang = double(pos) * pow(double(base), -2.0 * p / dh);
  tab[i] = make_float2(float(cos(ang)), float(sin(ang)));
}

__global__ __launch_bounds__(BT) void qkv_post_kernel(const float* __restrict__ qkv,
                                                      const float* __restrict__ b, int64_t T,
                                                      int S, int H, int Hkv, int dh,
                                                      const float* __restrict__ sa,
                                                      const float2* __restrict__ tab,
                                                      float* __restrict__ Qt, float* __restrict__ Kt,
                                                      float* __restrict__ Vv) {
  const int half = dh / 2;
  const int64_t W = int64_t(H + 2 * Hkv) * dh;
  const int64_t per_tok = int64_t(H + 2 * Hkv) * half;
  const int64_t i = int64_t(blockIdx.x) * BT + threadIdx.x;
  if (i >= T * per_tok) return;
  const int64_t t = i / per_tok;
  const int64_t j = i % per_tok;
  const int head = int(j / half), p = int(j % half);
  const float* row = qkv + t * W;
  if (head < H + Hkv) {
    const bool isq = head < H;
    const int64_t c0 = int64_t(head) * dh + p, c1 = c0 + half;
    float a = row[c0], bb = row[c1];
    if (b) {
      a += b[c0];
      bb += b[c1];
    }
    const float2 cssn = tab[(t % S) * half + p];
    const float cs = cssn.x, sn = cssn.y;
    const float ra = a * cs - bb * sn, rb = bb * cs + a * sn;
    if (isq) {
      const int g = head / (H / Hkv);
      const float s0 = sa ? sa[g * dh + p] : 1.0f, s1 = sa ? sa[g * dh + p + half] : 1.0f;
      Qt[t * int64_t(H) * dh + c0] = ra / s0;
      Qt[t * int64_t(H) * dh + c1] = rb / s1;
    } else {
      const int g = head - H;
      const float s0 = sa ? sa[g * dh + p] : 1.0f, s1 = sa ? sa[g * dh + p + half] : 1.0f;
      const int64_t k0 = t * int64_t(Hkv) * dh + int64_t(g) * dh + p;
      Kt[k0] = ra * s0;
      Kt[k0 + half] = rb * s1;
    }
  } else {
    const int g = head - H - Hkv;
    const int64_t c0 = int64_t(head) * dh + 2 * p;
    const int64_t v0 = t * int64_t(Hkv) * dh + int64_t(g) * dh + 2 * p;
    Vv[v0] = row[c0] + (b ? b[c0] : 0.0f);
    Vv[v0 + 1] = row[c0 + 1] + (b ? b[c0 + 1] : 0.0f);
  }
}

// Backward of qkv_post: dQ~, dK~, dV (w.r.t. Q~, K~, V) -> dQKV [T, (H + 2 Hkv) d]
// bf16 (the operand of the q/k/v gradient products): dq = RoPE^-1(dQ~ / s_a),
// dk = RoPE^-1(dK~ * s_a), dv = dV.  The bias gradient is the column sum of dQKV.
__global__ __launch_bounds__(BT) void qkv_post_bwd_kernel(const float* __restrict__ dQt,
                                                          const float* __restrict__ dKt,
                                                          const float* __restrict__ dV, int64_t T,
                                                          int S, int H, int Hkv, int dh,
                                                          const float* __restrict__ sa,
                                                          const float2* __restrict__ tab,
                                                          uint16_t* __restrict__ dqkv) {
  const int half = dh / 2;
  const int64_t W = int64_t(H + 2 * Hkv) * dh;
  const int64_t per_tok = int64_t(H + 2 * Hkv) * half;
  const int64_t i = int64_t(blockIdx.x) * BT + threadIdx.x;
  if (i >= T * per_tok) return;
  const int64_t t = i / per_tok;
  const int64_t j = i % per_tok;
  const int head = int(j / half), p = int(j % half);
  uint16_t* row = dqkv + t * W;
  if (head < H + Hkv) {
    const bool isq = head < H;
    float ga, gb;
    if (isq) {
      const int g = head / (H / Hkv);
      const float s0 = sa ? sa[g * dh + p] : 1.0f, s1 = sa ? sa[g * dh + p + half] : 1.0f;
      const int64_t q0 = t * int64_t(H) * dh + int64_t(head) * dh + p;
      ga = dQt[q0] / s0;
      gb = dQt[q0 + half] / s1;
    } else {
      const int g = head - H;
      const float s0 = sa ? sa[g * dh + p] : 1.0f, s1 = sa ? sa[g * dh + p + half] : 1.0f;
      const int64_t k0 = t * int64_t(Hkv) * dh + int64_t(g) * dh + p;
      ga = dKt[k0] * s0;
      gb = dKt[k0 + half] * s1;
    }
    const float2 cssn = tab[(t % S) * half + p];
    const float cs = cssn.x, sn = cssn.y;
    // the transpose of the rotation [[c, -s], [s, c]]
    const int64_t c0 = int64_t(head) * dh + p;
    row[c0] = f2bf(ga * cs + gb * sn);
    row[c0 + half] = f2bf(gb * cs - ga * sn);
  } else {
    const int g = head - H - Hkv;
    const int64_t c0 = int64_t(head) * dh + 2 * p;
    const int64_t v0 = t * int64_t(Hkv) * dh + int64_t(g) * dh + 2 * p;
    row[c0] = f2bf(dV[v0]);
    row[c0 + 1] = f2bf(dV[v0 + 1]);
  }
}

// ds_a[g d + c] = (sum_t dK~ K~ [.., g d + c] - sum over the group's query
// heads h of sum_t dQ~ Q~ [.., h d + c]) / s_a, from the column partials the
// activation backward wrote ([nq, H d] and [nk, Hkv d]), in fixed order.
// Workgroup: 64 channels x 16 row slices; each thread sums its slice's rows in
// order (fp64), the slices combine in a fixed tree: deterministic.
constexpr int SA_COLS = 64, SA_SLICES = 16;
__global__ __launch_bounds__(SA_COLS * SA_SLICES) void sa_grad_finish_kernel(
    const float* __restrict__ pq, int64_t nq, const float* __restrict__ pk, int64_t nk, int H,
    int Hkv, int dh, const float* __restrict__ sa, float* __restrict__ dsa) {
  __shared__ double red[SA_SLICES][SA_COLS];
  const int tc = threadIdx.x % SA_COLS, ts = threadIdx.x / SA_COLS;
  const int64_t c = int64_t(blockIdx.x) * SA_COLS + tc;
  const int64_t Ck = int64_t(Hkv) * dh, Cq = int64_t(H) * dh;
  double acc = 0.0;
  if (c < Ck) {
    const int g = int(c / dh), e = int(c % dh);
    for (int64_t i = ts; i < nk; i += SA_SLICES) acc += double(pk[i * Ck + c]);
    const int grp = H / Hkv;
    for (int hq = g * grp; hq < (g + 1) * grp; ++hq)
      for (int64_t i = ts; i < nq; i += SA_SLICES) acc -= double(pq[i * Cq + int64_t(hq) * dh + e]);
  }
  red[ts][tc] = acc;
  __syncthreads();
  for (int w = SA_SLICES / 2; w > 0; w >>= 1) {
    if (ts < w) red[ts][tc] += red[ts + w][tc];
    __syncthreads();
  }
  if (ts == 0 && c < Ck) dsa[c] = float(red[0][tc] / double(sa[c]));
}

// ------------------------------------------------------------------ SiLU gating
// GU [T, 2F] fp32 (gate | up) plus bias -> x4 = SiLU(gate) * up (fp32); the
// biased GU kept in place for the backward.
__global__ __launch_bounds__(BT) void silu_mul_kernel(float* __restrict__ gu,
                                                      const float* __restrict__ b, int64_t T,
                                                      int64_t F, float* __restrict__ x4) {
  const int64_t i = int64_t(blockIdx.x) * BT + threadIdx.x;
  if (i >= T * F) return;
  const int64_t t = i / F, c = i % F;
  float g = gu[t * 2 * F + c], u = gu[t * 2 * F + F + c];
  if (b) {
    g += b[c];
    u += b[F + c];
    gu[t * 2 * F + c] = g;
    gu[t * 2 * F + F + c] = u;
  }
  const float sg = 1.0f / (1.0f + expf(-g));
  x4[i] = g * sg * u;
}

// dGU (bf16 operand) from dx4: dgate = dx4 * up * sg (1 + g (1 - sg)), dup = dx4 * g sg.
__global__ __launch_bounds__(BT) void silu_mul_bwd_kernel(const float* __restrict__ gu,
                                                          const float* __restrict__ dx4, int64_t T,
                                                          int64_t F, uint16_t* __restrict__ dgu) {
  const int64_t i = int64_t(blockIdx.x) * BT + threadIdx.x;
  if (i >= T * F) return;
  const int64_t t = i / F, c = i % F;
  const float g = gu[t * 2 * F + c], u = gu[t * 2 * F + F + c];
  const float sg = 1.0f / (1.0f + expf(-g));
  const float d = dx4[i];
  dgu[t * 2 * F + c] = f2bf(d * u * (sg * (1.0f + g * (1.0f - sg))));
  dgu[t * 2 * F + F + c] = f2bf(d * (g * sg));
}

// ------------------------------------------------------------------ residual, loss
// out = base + y + b[c] (base fp32 or bf16).
template <typename TB>
__global__ __launch_bounds__(BT) void resid_add_kernel(const TB* __restrict__ base,
                                                       const float* __restrict__ y,
                                                       const float* __restrict__ b, int64_t T,
                                                       int64_t D, float* __restrict__ out) {
  const int64_t i = int64_t(blockIdx.x) * BT + threadIdx.x;
  if (i >= T * D) return;
  out[i] = load1(base + i) + y[i] + (b ? b[i % D] : 0.0f);
}

// Per token row: R = h2 - target; row partial sum of R^2 (fp64); dh2 = R *
// scale (fp32, and bf16 for the products).
__global__ __launch_bounds__(BT) void block_loss_kernel(const float* __restrict__ h2,
                                                        const uint16_t* __restrict__ tgt, int64_t D,
                                                        float scale, float* __restrict__ dh,
                                                        uint16_t* __restrict__ dh16,
                                                        double* __restrict__ rows) {
  __shared__ double sh[4];
  const int64_t row = blockIdx.x;
  double s = 0.0;
  for (int64_t c = threadIdx.x; c < D; c += BT) {
    const int64_t i = row * D + c;
    const float r = h2[i] - bf2f(tgt[i]);
    s += double(r) * double(r);
    const float g = r * scale;
    dh[i] = g;
    dh16[i] = f2bf(g);
  }
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) s += __shfl_xor(s, off);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh[w] = s;
  __syncthreads();
  if (threadIdx.x == 0) rows[row] = ((sh[0] + sh[1]) + sh[2]) + sh[3];
}

__global__ __launch_bounds__(1024) void sum_rows_kernel(const double* __restrict__ rows, int64_t n,
                                                        double inv_n, float* __restrict__ loss) {
  __shared__ double sh[16];
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += 1024) s += rows[i];
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) s += __shfl_xor(s, off);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh[w] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (int k = 0; k < 16; ++k) t += sh[k];
    *loss = float(t * inv_n);
  }
}

// out (bf16) = in (fp32) / s[c] (s null: a plain conversion).
__global__ __launch_bounds__(BT) void scale_to_bf16_kernel(const float* __restrict__ in,
                                                           const float* __restrict__ s, int64_t T,
                                                           int64_t C, uint16_t* __restrict__ out) {
  const int64_t i = int64_t(blockIdx.x) * BT + threadIdx.x;
  if (i >= T * C) return;
  out[i] = f2bf(s ? in[i] / s[i % C] : in[i]);
}

unsigned blocks_for(int64_t n) { return unsigned((n + BT - 1) / BT); }

}  // namespace

hipError_t rmsnorm_fwd(const void* h, bool h_bf16, const float* g, int64_t T, int64_t D, float eps,
                       float* x, float* rstd, hipStream_t st) {
  if (T <= 0) return hipSuccess;
  if (h_bf16)
    hipLaunchKernelGGL(rmsnorm_fwd_kernel<uint16_t>, dim3(unsigned(T)), dim3(BT), 0, st,
                       static_cast<const uint16_t*>(h), g, D, eps, x, rstd);
  else
    hipLaunchKernelGGL(rmsnorm_fwd_kernel<float>, dim3(unsigned(T)), dim3(BT), 0, st,
                       static_cast<const float*>(h), g, D, eps, x, rstd);
  return hipGetLastError();
}

hipError_t rmsnorm_bwd(const void* h, bool h_bf16, const float* g, const float* rstd,
                       const float* dxt, const float* s, const float* dres, int64_t T, int64_t D,
                       float* dh, hipStream_t st) {
  if (T <= 0) return hipSuccess;
  if (h_bf16)
    hipLaunchKernelGGL(rmsnorm_bwd_kernel<uint16_t>, dim3(unsigned(T)), dim3(BT), 0, st,
                       static_cast<const uint16_t*>(h), g, rstd, dxt, s, dres, D, dh);
  else
    hipLaunchKernelGGL(rmsnorm_bwd_kernel<float>, dim3(unsigned(T)), dim3(BT), 0, st,
                       static_cast<const float*>(h), g, rstd, dxt, s, dres, D, dh);
  return hipGetLastError();
}

hipError_t rope_table(int S, int dh, float base, float* tab, hipStream_t st) {
  const int64_t n = int64_t(S) * (dh / 2);
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(rope_table_kernel, dim3(blocks_for(n)), dim3(BT), 0, st, S, dh, base,
                     reinterpret_cast<float2*>(tab));
  return hipGetLastError();
}

hipError_t qkv_post(const float* qkv, const float* b, int64_t T, int S, int H, int Hkv, int dh,
                    const float* tab, const float* sa, float* Qt, float* Kt, float* V,
                    hipStream_t st) {
  const int64_t n = T * int64_t(H + 2 * Hkv) * (dh / 2);
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(qkv_post_kernel, dim3(blocks_for(n)), dim3(BT), 0, st, qkv, b, T, S, H, Hkv,
                     dh, sa, reinterpret_cast<const float2*>(tab), Qt, Kt, V);
  return hipGetLastError();
}

hipError_t qkv_post_bwd(const float* dQt, const float* dKt, const float* dV, int64_t T, int S,
                        int H, int Hkv, int dh, const float* tab, const float* sa, void* dqkv,
                        hipStream_t st) {
  const int64_t n = T * int64_t(H + 2 * Hkv) * (dh / 2);
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(qkv_post_bwd_kernel, dim3(blocks_for(n)), dim3(BT), 0, st, dQt, dKt, dV, T,
                     S, H, Hkv, dh, sa, reinterpret_cast<const float2*>(tab),
                     static_cast<uint16_t*>(dqkv));
  return hipGetLastError();
}

hipError_t sa_grad_finish(const float* pq, int64_t nq, const float* pk, int64_t nk, int H, int Hkv,
                          int dh, const float* sa, float* dsa, hipStream_t st) {
  const int64_t n = int64_t(Hkv) * dh;
  hipLaunchKernelGGL(sa_grad_finish_kernel, dim3(unsigned((n + SA_COLS - 1) / SA_COLS)),
                     dim3(SA_COLS * SA_SLICES), 0, st, pq, nq, pk, nk, H, Hkv, dh, sa, dsa);
  return hipGetLastError();
}

hipError_t silu_mul(float* gu, const float* b, int64_t T, int64_t F, float* x4, hipStream_t st) {
  if (T * F <= 0) return hipSuccess;
  hipLaunchKernelGGL(silu_mul_kernel, dim3(blocks_for(T * F)), dim3(BT), 0, st, gu, b, T, F, x4);
  return hipGetLastError();
}

hipError_t silu_mul_bwd(const float* gu, const float* dx4, int64_t T, int64_t F, void* dgu,
                        hipStream_t st) {
  if (T * F <= 0) return hipSuccess;
  hipLaunchKernelGGL(silu_mul_bwd_kernel, dim3(blocks_for(T * F)), dim3(BT), 0, st, gu, dx4, T, F,
                     static_cast<uint16_t*>(dgu));
  return hipGetLastError();
}

hipError_t resid_add(const void* base, bool base_bf16, const float* y, const float* b, int64_t T,
                     int64_t D, float* out, hipStream_t st) {
  if (T * D <= 0) return hipSuccess;
  if (base_bf16)
    hipLaunchKernelGGL(resid_add_kernel<uint16_t>, dim3(blocks_for(T * D)), dim3(BT), 0, st,
                       static_cast<const uint16_t*>(base), y, b, T, D, out);
  else
    hipLaunchKernelGGL(resid_add_kernel<float>, dim3(blocks_for(T * D)), dim3(BT), 0, st,
                       static_cast<const float*>(base), y, b, T, D, out);
  return hipGetLastError();
}

hipError_t block_loss(const float* h2, const void* tgt, int64_t T, int64_t D, float* dh,
                      void* dh16, double* rows, float* loss, hipStream_t st) {
  if (T <= 0) return hipSuccess;
  const double n = double(T) * double(D);
  hipLaunchKernelGGL(block_loss_kernel, dim3(unsigned(T)), dim3(BT), 0, st, h2,
                     static_cast<const uint16_t*>(tgt), D, float(2.0 / n), dh,
                     static_cast<uint16_t*>(dh16), rows);
  hipLaunchKernelGGL(sum_rows_kernel, dim3(1), dim3(1024), 0, st, rows, T, 1.0 / n, loss);
  return hipGetLastError();
}

hipError_t scale_to_bf16(const float* in, const float* s, int64_t T, int64_t C, void* out,
                         hipStream_t st) {
  if (T * C <= 0) return hipSuccess;
  hipLaunchKernelGGL(scale_to_bf16_kernel, dim3(blocks_for(T * C)), dim3(BT), 0, st, in, s, T, C,
                     static_cast<uint16_t*>(out));
  return hipGetLastError();
}

}  // namespace oq

namespace oq {
namespace {
__global__ __launch_bounds__(256) void colsum_finish_kernel(const double* __restrict__ parts,
                                                            int64_t n, int64_t C,
                                                            float* __restrict__ out) {
  const int64_t c = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (c >= C) return;
  double s = 0.0;
  for (int64_t i = 0; i < n; ++i) s += parts[i * C + c];
  out[c] = float(s);
}
}  // namespace

// out[c] = sum over the n partial rows (fp64, in order), rounded once.
hipError_t colsum_finish(const double* parts, int64_t n, int64_t C, float* out, hipStream_t st) {
  if (C <= 0) return hipSuccess;
  hipLaunchKernelGGL(colsum_finish_kernel, dim3(unsigned((C + 255) / 256)), dim3(256), 0, st, parts,
                     n, C, out);
  return hipGetLastError();
}
}  // namespace oq
