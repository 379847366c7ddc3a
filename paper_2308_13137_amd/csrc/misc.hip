// Bandwidth-bound helpers of the calibration step: tiled transposes, the LET
// bias fold, column reductions with fixed-order finishing passes, the loss
// reduction and the AdamW update.  Every reduction is a fixed tree (wave
// butterflies, then ordered loops), never atomics, so results are bitwise
// reproducible.
#include <math.h>

#include <algorithm>
#include <cmath>

#include "common.h"
#include "oq_internal.h"

namespace oq {
namespace {

// ------------------------------------------------------------------ transpose
// out[c][r] = in[r][c]; 64x64 tiles through LDS, 256 threads, 16 elements each.
template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(const T* __restrict__ in, int64_t rows,
                                                        int64_t cols, int64_t ld_in,
                                                        T* __restrict__ out, int64_t ld_out) {
  __shared__ T tile[64][65];
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int64_t r0 = int64_t(blockIdx.y) * 64, c0 = int64_t(blockIdx.x) * 64;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int r = ty + 4 * i;
    if (r0 + r < rows && c0 + tx < cols) tile[r][tx] = in[(r0 + r) * ld_in + c0 + tx];
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int c = ty + 4 * i;
    if (c0 + c < cols && r0 + tx < rows) out[(c0 + c) * ld_out + r0 + tx] = tile[tx][c];
  }
}

// ------------------------------------------------------------------ LET fold
// One wave per output row: B~[o] = B[o] + sum_c W[o,c] delta[c] (fp64 sum),
// W~[o,c] = W[o,c] * s[c].
template <typename TW, typename TT>
__global__ __launch_bounds__(256) void let_fold_kernel(const TW* __restrict__ W, const float* B,
                                                       int64_t c_out, int64_t c_in,
                                                       const float* s, const float* delta,
                                                       TT* Wt, float* Bt) {
  const int lane = threadIdx.x & 63;
  const int64_t o = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (o >= c_out) return;
  const int64_t cpr = c_in / 8;
  double acc = 0.0;
  for (int64_t j = lane; j < cpr; j += 64) {
    float w[8];
    load8(W + o * c_in + 8 * j, w);
    if (delta) {
      float d[8];
      load8(delta + 8 * j, d);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc += double(w[e]) * double(d[e]);
    }
    if (Wt) {
      float sv[8], t[8];
      if (s) load8(s + 8 * j, sv);
#pragma unroll
      for (int e = 0; e < 8; ++e) t[e] = s ? w[e] * sv[e] : w[e];
      store8(Wt + o * c_in + 8 * j, t);
    }
  }
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) acc += __shfl_xor(acc, off);
  if (lane == 0 && Bt) Bt[o] = float(acc + (B ? double(B[o]) : 0.0));
}

// ------------------------------------------------------------------ LET absorption
// Folds a site's LET into the op that produces its input: row c of P [C, n]
// (a normalisation's gain is n = 1, a previous linear's weight has its output
// channels as rows) becomes P[c, :] * (1/s[c]) and its bias (b[c] - delta[c])
// * (1/s[c]), the same fp32 order as the activation transform (x - delta)*(1/s).
template <typename TP>
__global__ __launch_bounds__(256) void let_absorb_kernel(const TP* __restrict__ P,
                                                         const float* __restrict__ b, int64_t C,
                                                         int64_t n, const float* __restrict__ s,
                                                         const float* __restrict__ delta,
                                                         TP* __restrict__ Pout,
                                                         float* __restrict__ bout) {
  const int64_t total = C * n;
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < total;
       i += int64_t(gridDim.x) * 256) {
    const int64_t c = i / n;
    const float r = s ? div_rn(1.0f, s[c]) : 1.0f;
    if (Pout) store1(Pout + i, load1(P + i) * r);
    if (bout && i % n == 0) {
      const float bb = b ? b[c] : 0.0f;
      bout[c] = (delta ? bb - delta[c] : bb) * r;
    }
  }
}

// ------------------------------------------------------------------ column reductions
// Grid (column tiles of 2048, row blocks of R rows); thread owns 8 columns.
template <typename TW>
__global__ __launch_bounds__(256) void wcolsum_kernel(const TW* __restrict__ W, int64_t rows,
                                                      int64_t cols, int R, const float* wt,
                                                      float* out_parts) {
  const int64_t c = (int64_t(blockIdx.x) * 256 + threadIdx.x) * 8;
  if (c >= cols) return;
  const int64_t r0 = int64_t(blockIdx.y) * R, r1 = min(rows, r0 + R);
  float acc[8] = {};
  for (int64_t r = r0; r < r1; ++r) {
    float w[8];
    load8(W + r * cols + c, w);
    const float f = wt[r];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += f * w[e];
  }
  store8(out_parts + int64_t(blockIdx.y) * cols + c, acc);
}

template <typename TX>
__global__ __launch_bounds__(256) void colstat_kernel(const TX* __restrict__ X, int64_t rows,
                                                      int64_t cols, int R, float* amax_parts,
                                                      double* sum_parts) {
  const int64_t c = (int64_t(blockIdx.x) * 256 + threadIdx.x) * 8;
  if (c >= cols) return;
  const int64_t r0 = int64_t(blockIdx.y) * R, r1 = min(rows, r0 + R);
  float mx[8] = {};
  double sm[8] = {};
  for (int64_t r = r0; r < r1; ++r) {
    float x[8];
    load8(X + r * cols + c, x);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      mx[e] = fmaxf(mx[e], fabsf(x[e]));
      sm[e] += double(x[e]);
    }
  }
  store8(amax_parts + int64_t(blockIdx.y) * cols + c, mx);
  if (sum_parts) {
#pragma unroll
    for (int e = 0; e < 8; ++e) sum_parts[int64_t(blockIdx.y) * cols + c + e] = sm[e];
  }
}

// Column sums of [rows, C] partial arrays: a block of 16 waves covers 64
// columns (lane = column); wave w adds rows w, w + 16, ... in fp64 into four
// accumulators (four loads in flight; row w + 16 k goes to accumulator
// k % 4), and the 16 wave sums are combined through LDS in wave order.  Every
// order is fixed, so the result is deterministic.
constexpr int CS_WAVES = 16;

OQ_DEV double strip_sum(const float* parts, int64_t rows, int64_t C, int64_t c, int w) {
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  if (parts && c < C) {
    int64_t i = w;
    for (; i + 3 * CS_WAVES < rows; i += 4 * CS_WAVES) {
      float v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = parts[(i + u * CS_WAVES) * C + c];
#pragma unroll
      for (int u = 0; u < 4; ++u) acc[u] += double(v[u]);
    }
#pragma unroll
    for (int u = 0; u < 3; ++u)
      if (i + u * CS_WAVES < rows) acc[u] += double(parts[(i + u * CS_WAVES) * C + c]);
  }
  return (acc[0] + acc[1]) + (acc[2] + acc[3]);
}

template <int NA>
OQ_DEV void strip_combine(double (&v)[NA], double (*sh)[CS_WAVES][64], int w, int lane) {
#pragma unroll
  for (int a = 0; a < NA; ++a) sh[a][w][lane] = v[a];
  __syncthreads();
#pragma unroll
  for (int a = 0; a < NA; ++a) {
    double r = 0.0;
    for (int k = 0; k < CS_WAVES; ++k) r += sh[a][k][lane];
    v[a] = r;
  }
}

__global__ __launch_bounds__(64 * CS_WAVES) void let_grad_finish_kernel(
    int64_t C, const float* s, const float* pw, int64_t npw, const float* psx, const float* ps1,
    int64_t npa, const float* pb, int64_t npb, float* d_s, float* d_delta) {
  __shared__ double sh[4][CS_WAVES][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t c = int64_t(blockIdx.x) * 64 + lane;
  double v[4] = {strip_sum(pw, npw, C, c, w), strip_sum(psx, npa, C, c, w),
                 strip_sum(ps1, npa, C, c, w), strip_sum(pb, npb, C, c, w)};
  strip_combine<4>(v, sh, w, lane);
  if (w != 0 || c >= C) return;
  const double sc = s ? double(s[c]) : 1.0;
  if (d_s) d_s[c] = float(v[0] - v[1] / sc);
  if (d_delta) d_delta[c] = float(v[3] - v[2] / sc);
}

__global__ __launch_bounds__(64 * CS_WAVES) void let_init_finish_kernel(
    int64_t C, int64_t T, const float* ax_parts, int64_t nax, const double* sum_parts,
    const float* aw_parts, int64_t naw, float* s, float* delta) {
  __shared__ double sh[1][CS_WAVES][64];
  __shared__ float shm[2][CS_WAVES][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t c = int64_t(blockIdx.x) * 64 + lane;
  float ax = 0.f, aw = 0.f;
  double v[1] = {0.0};
  if (c < C) {
    for (int64_t i = w; i < nax; i += CS_WAVES) {
      ax = fmaxf(ax, ax_parts[i * C + c]);
      v[0] += sum_parts[i * C + c];
    }
    for (int64_t i = w; i < naw; i += CS_WAVES) aw = fmaxf(aw, aw_parts[i * C + c]);
  }
  shm[0][w][lane] = ax;
  shm[1][w][lane] = aw;
  strip_combine<1>(v, sh, w, lane);
  if (w != 0 || c >= C) return;
  for (int k = 0; k < CS_WAVES; ++k) {
    ax = fmaxf(ax, shm[0][k][lane]);
    aw = fmaxf(aw, shm[1][k][lane]);
  }
  ax = fmaxf(ax, 1e-5f);
  aw = fmaxf(aw, 1e-5f);
  s[c] = div_rn(sqrt_rn(ax), sqrt_rn(aw));
  delta[c] = float(v[0] / double(T));
}

// ------------------------------------------------------------------ loss
// One wave per row: fp64 sums of the per-column-tile partials.
__global__ __launch_bounds__(256) void row_partials_kernel(const float* __restrict__ psq,
                                                           const float* __restrict__ pdy,
                                                           int64_t M, int ntn, double* rl,
                                                           float* dbt) {
  const int lane = threadIdx.x & 63;
  const int64_t m = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (m >= M) return;
  double a = 0.0, b = 0.0;
  for (int j = lane; j < ntn; j += 64) {
    a += double(psq[m * ntn + j]);
    if (pdy) b += double(pdy[m * ntn + j]);
  }
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    a += __shfl_xor(a, off);
    b += __shfl_xor(b, off);
  }
  if (lane == 0) {
    rl[m] = a;
    if (pdy && dbt) dbt[m] = float(b);
  }
}

// One block of 16 waves; thread t adds rows t, t + 1024, ... of each linear
// into four accumulators (row t + 1024 k goes to accumulator k % 4), then
// the wave and the 16 waves combine in a fixed order.
__global__ __launch_bounds__(1024) void loss_finish_kernel(const double* rl, LossArgs la,
                                                           float* loss) {
  __shared__ double sh[16];
  const int tid = threadIdx.x;
  double total = 0.0;
  for (int l = 0; l < la.nlin; ++l) {
    const int64_t b = la.row_begin[l], e = la.row_end[l];
    float* out = la.row_loss[l];
    double a[4] = {0.0, 0.0, 0.0, 0.0};
    int64_t m = b + tid;
    for (; m + 3 * 1024 < e; m += 4 * 1024) {
      double v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = rl[m + u * 1024];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        a[u] += v[u];
        if (out) out[m + u * 1024 - b] = float(v[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < 3; ++u) {
      const int64_t mu = m + u * 1024;
      if (mu < e) {
        a[u] += rl[mu];
        if (out) out[mu - b] = float(rl[mu]);
      }
    }
    double s = (a[0] + a[1]) + (a[2] + a[3]);
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) s += __shfl_xor(s, off);
    __syncthreads();
    if ((tid & 63) == 0) sh[tid >> 6] = s;
    __syncthreads();
    double r = 0.0;
#pragma unroll
    for (int w = 0; w < 16; ++w) r += sh[w];
    total += r * la.inv_n[l];
  }
  if (tid == 0) *loss = float(total);
}

// ------------------------------------------------------------------ AdamW
__global__ __launch_bounds__(256) void adamw_kernel(float* p, const float* g, float* m, float* v,
                                                    int64_t n, AdamCoef c) {
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (i >= n) return;
  const float gi = g[i];
  const float mi = c.b1 * m[i] + c.omb1 * gi;
  const float vi = c.b2 * v[i] + c.omb2 * (gi * gi);
  m[i] = mi;
  v[i] = vi;
  const float mh = mi / c.bc1;
  const float vh = vi / c.bc2;
  p[i] = p[i] * c.decay - c.lr * (mh / (__fsqrt_rn(vh) + c.eps));
}

// Several tensors in one launch: block b belongs to the tensor whose block
// range holds it (at most ADAM_MAX tensors, two coefficient sets).
__global__ __launch_bounds__(256) void adamw_multi_kernel(AdamList L, AdamCoef c0, AdamCoef c1) {
  int k = 0;
#pragma unroll 1
  while (k + 1 < L.n && int(blockIdx.x) >= L.block_begin[k + 1]) ++k;
  const AdamCoef& c = L.set[k] ? c1 : c0;
  const int64_t i = int64_t(blockIdx.x - L.block_begin[k]) * 256 + threadIdx.x;
  if (i >= L.len[k]) return;
  float* p = L.p[k];
  float* m = L.m[k];
  float* v = L.v[k];
  const float gi = L.g[k][i];
  const float mi = c.b1 * m[i] + c.omb1 * gi;
  const float vi = c.b2 * v[i] + c.omb2 * (gi * gi);
  m[i] = mi;
  v[i] = vi;
  const float mh = mi / c.bc1;
  const float vh = vi / c.bc2;
  p[i] = p[i] * c.decay - c.lr * (mh / (__fsqrt_rn(vh) + c.eps));
}

// ------------------------------------------------------------------ K-split partial sums
// d[i] = ((c[i] + c[i + stride]) + c[i + 2 stride]) + ...  (fixed order); d
// may be c (in place over the first partial); grid stride, four elements per
// thread when the layout allows.
__global__ __launch_bounds__(256) void sum_partials4_kernel(const float* c, float* d, int64_t n4,
                                                            int parts, int64_t stride4) {
  const float4* c4 = reinterpret_cast<const float4*>(c);
  float4* d4 = reinterpret_cast<float4*>(d);
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n4;
       i += int64_t(gridDim.x) * 256) {
    float4 a = c4[i];
    for (int s = 1; s < parts; ++s) {
      const float4 b = c4[i + s * stride4];
      a.x += b.x;
      a.y += b.y;
      a.z += b.z;
      a.w += b.w;
    }
    d4[i] = a;
  }
}

__global__ __launch_bounds__(256) void sum_partials1_kernel(const float* c, float* d, int64_t n,
                                                            int parts, int64_t stride) {
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * 256) {
    float a = c[i];
    for (int s = 1; s < parts; ++s) a += c[i + s * stride];
    d[i] = a;
  }
}

}  // namespace

hipError_t transpose(const void* in, int64_t rows, int64_t cols, int64_t ld_in, void* out,
                     int64_t ld_out, int elem_bytes, hipStream_t st) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  const int64_t gy = (rows + 63) / 64, gx = (cols + 63) / 64;
  if (gy > 65535 || gx > 0x7fffffff) return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(gx), static_cast<unsigned>(gy));
  if (elem_bytes == 2)
    hipLaunchKernelGGL(transpose_kernel<uint16_t>, grid, dim3(256), 0, st,
                       static_cast<const uint16_t*>(in), rows, cols, ld_in,
                       static_cast<uint16_t*>(out), ld_out);
  else if (elem_bytes == 4)
    hipLaunchKernelGGL(transpose_kernel<float>, grid, dim3(256), 0, st,
                       static_cast<const float*>(in), rows, cols, ld_in, static_cast<float*>(out),
                       ld_out);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t let_fold(const void* W, bool w_bf16, const float* B, int64_t c_out, int64_t c_in,
                    const float* s, const float* delta, void* Wt, bool wt_bf16, float* Bt,
                    hipStream_t st) {
  if (c_out <= 0) return hipSuccess;
  const dim3 grid(unsigned((c_out + 3) / 4));
  auto go = [&](auto tw, auto tt) {
    using TW = decltype(tw);
    using TT = decltype(tt);
    hipLaunchKernelGGL((let_fold_kernel<TW, TT>), grid, dim3(256), 0, st,
                       static_cast<const TW*>(W), B, c_out, c_in, s, delta, static_cast<TT*>(Wt),
                       Bt);
  };
  if (w_bf16) {
    if (wt_bf16) go(uint16_t{}, uint16_t{}); else go(uint16_t{}, float{});
  } else {
    if (wt_bf16) go(float{}, uint16_t{}); else go(float{}, float{});
  }
  return hipGetLastError();
}

hipError_t let_absorb(const void* P, bool p_bf16, const float* b, int64_t C, int64_t n,
                      const float* s, const float* delta, void* Pout, float* bout,
                      hipStream_t st) {
  if (C <= 0 || n <= 0) return hipSuccess;
  const dim3 grid(unsigned(std::min<int64_t>((C * n + 255) / 256, 4096)));
  if (p_bf16)
    hipLaunchKernelGGL((let_absorb_kernel<uint16_t>), grid, dim3(256), 0, st,
                       static_cast<const uint16_t*>(P), b, C, n, s, delta,
                       static_cast<uint16_t*>(Pout), bout);
  else
    hipLaunchKernelGGL((let_absorb_kernel<float>), grid, dim3(256), 0, st,
                       static_cast<const float*>(P), b, C, n, s, delta, static_cast<float*>(Pout),
                       bout);
  return hipGetLastError();
}

static int64_t colred_rows(int64_t rows) { return std::max<int64_t>(16, (rows + 511) / 512); }

int64_t wcolsum_nparts(int64_t rows) {
  if (rows <= 0) return 0;
  const int64_t R = colred_rows(rows);
  return (rows + R - 1) / R;
}

hipError_t wcolsum(const void* W, bool w_bf16, int64_t rows, int64_t cols, const float* wt,
                   float* out_parts, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  const int64_t R = colred_rows(rows);
  const dim3 grid(unsigned((cols / 8 + 255) / 256), unsigned((rows + R - 1) / R));
  if (w_bf16)
    hipLaunchKernelGGL(wcolsum_kernel<uint16_t>, grid, dim3(256), 0, st,
                       static_cast<const uint16_t*>(W), rows, cols, int(R), wt, out_parts);
  else
    hipLaunchKernelGGL(wcolsum_kernel<float>, grid, dim3(256), 0, st,
                       static_cast<const float*>(W), rows, cols, int(R), wt, out_parts);
  return hipGetLastError();
}

int64_t colstat_nparts(int64_t rows) { return wcolsum_nparts(rows); }

hipError_t colstat(const void* X, bool bf16, int64_t rows, int64_t cols, float* amax_parts,
                   double* sum_parts, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  const int64_t R = colred_rows(rows);
  const dim3 grid(unsigned((cols / 8 + 255) / 256), unsigned((rows + R - 1) / R));
  if (bf16)
    hipLaunchKernelGGL(colstat_kernel<uint16_t>, grid, dim3(256), 0, st,
                       static_cast<const uint16_t*>(X), rows, cols, int(R), amax_parts, sum_parts);
  else
    hipLaunchKernelGGL(colstat_kernel<float>, grid, dim3(256), 0, st,
                       static_cast<const float*>(X), rows, cols, int(R), amax_parts, sum_parts);
  return hipGetLastError();
}

hipError_t let_grad_finish(int64_t C, const float* s, const float* pw, int64_t npw,
                           const float* psx, const float* ps1, int64_t npa, const float* pb,
                           int64_t npb, float* d_s, float* d_delta, hipStream_t st) {
  if (C <= 0) return hipSuccess;
  hipLaunchKernelGGL(let_grad_finish_kernel, dim3(unsigned((C + 63) / 64)), dim3(64 * CS_WAVES), 0, st, C,
                     s, pw, npw, psx, ps1, npa, pb, npb, d_s, d_delta);
  return hipGetLastError();
}

hipError_t let_init_finish(int64_t C, int64_t T, const float* ax_parts, int64_t nax,
                           const double* sum_parts, const float* aw_parts, int64_t naw, float* s,
                           float* delta, hipStream_t st) {
  if (C <= 0) return hipSuccess;
  hipLaunchKernelGGL(let_init_finish_kernel, dim3(unsigned((C + 63) / 64)), dim3(64 * CS_WAVES), 0, st, C,
                     T, ax_parts, nax, sum_parts, aw_parts, naw, s, delta);
  return hipGetLastError();
}

hipError_t row_partials(const float* psq, const float* pdy, int64_t M, int ntn, double* rl,
                        float* dbt, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  hipLaunchKernelGGL(row_partials_kernel, dim3(unsigned((M + 3) / 4)), dim3(256), 0, st, psq, pdy,
                     M, ntn, rl, dbt);
  return hipGetLastError();
}

hipError_t loss_finish(const double* rl, LossArgs la, float* loss, hipStream_t st) {
  hipLaunchKernelGGL(loss_finish_kernel, dim3(1), dim3(1024), 0, st, rl, la, loss);
  return hipGetLastError();
}

AdamCoef adam_coef(double lr, double b1, double b2, double eps, double wd, int step) {
  AdamCoef c;
  c.lr = float(lr);
  c.b1 = float(b1);
  c.omb1 = float(1.0 - b1);
  c.b2 = float(b2);
  c.omb2 = float(1.0 - b2);
  c.eps = float(eps);
  c.decay = float(1.0 - lr * wd);
  c.bc1 = float(1.0 - std::pow(b1, double(step)));
  c.bc2 = float(1.0 - std::pow(b2, double(step)));
  return c;
}

hipError_t adamw_multi(const AdamList& L, AdamCoef c0, AdamCoef c1, hipStream_t st) {
  if (L.n <= 0) return hipSuccess;
  AdamList l = L;
  int blocks = 0;
  for (int k = 0; k < l.n; ++k) {
    l.block_begin[k] = blocks;
    const int64_t nb = (l.len[k] + 255) / 256;
    if (blocks + nb > (int64_t(1) << 31) - 1) return hipErrorInvalidValue;
    blocks += int(nb);
  }
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(adamw_multi_kernel, dim3(unsigned(blocks)), dim3(256), 0, st, l, c0, c1);
  return hipGetLastError();
}

hipError_t sum_partials_to(const float* c, float* d, int64_t n, int parts, int64_t stride,
                           hipStream_t st) {
  if (n <= 0) return hipSuccess;
  if (parts < 1 || (parts > 1 && stride < n)) return hipErrorInvalidValue;
  if (parts == 1 && c == d) return hipSuccess;
  const bool v4 = n % 4 == 0 && stride % 4 == 0 && (reinterpret_cast<uintptr_t>(c) & 15) == 0 &&
                  (reinterpret_cast<uintptr_t>(d) & 15) == 0;
  const int64_t work = v4 ? n / 4 : n;
  const unsigned grid = unsigned(std::min<int64_t>((work + 255) / 256, 8192));
  if (v4)
    hipLaunchKernelGGL(sum_partials4_kernel, dim3(grid), dim3(256), 0, st, c, d, n / 4, parts,
                       stride / 4);
  else
    hipLaunchKernelGGL(sum_partials1_kernel, dim3(grid), dim3(256), 0, st, c, d, n, parts, stride);
  return hipGetLastError();
}

hipError_t sum_partials(float* c, int64_t n, int parts, int64_t stride, hipStream_t st) {
  if (parts <= 1) return hipSuccess;
  return sum_partials_to(c, c, n, parts, stride, st);
}

hipError_t adamw(float* p, const float* g, float* m, float* v, int64_t n, AdamCoef c,
                 hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(adamw_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, st, p, g, m, v,
                     n, c);
  return hipGetLastError();
}

}  // namespace oq
