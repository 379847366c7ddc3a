// Causal multi-head attention for the whole-block calibration step (the
// attention operation of Sec. 3.3 with the quantised Q^, K^, V^ of Eq. 5),
// forward and backward, on bf16 matrix cores (v_mfma_f32_16x16x32_bf16).
//
// Layouts: Q^ [T, H d], K^ and V^ [T, Hkv d] bf16, token-major with the
// heads side by side (T = n_seq * S, the samples one after another); query
// head h reads key/value head h / (H / Hkv).  O and the gradients fp32 in
// the same layouts; the per-query softmax statistic LSE [H, T] is kept in
// base 2 of the scaled logits (t = s * log2(e) / sqrt(d)).
//
// Forward (one workgroup = 64 queries of one head, four waves of 16): each
// wave computes S^T = K Q^T for a 64-key tile (keys on the matrix rows), so
// a lane's accumulators all belong to one query: the online softmax needs
// only in-lane work and two cross-lane exchanges, and the probabilities feed
// the O^T = V^T P product as its B operand straight from registers (the
// k-order of the product is permuted to match: any consistent order of the
// summed index gives the same sum).  K is staged in LDS row-major (XOR
// swizzled chunks), V transposed (padded rows).
//
// Backward (deterministic, no atomics): one kernel per 64-key tile and key
// head accumulates dK, dV over every query tile and query head of its group
// (S^T, dP^T recomputed from LSE; P and dS staged per wave in LDS to become
// A operands); a second kernel per 64-query tile accumulates dQ over the key
// tiles, after a first sweep that forms D = sum_j P_ij dP_ij (written out for
// the dK/dV kernel, which runs after it).
//
// Rounding: P and dS enter the matrix cores as bf16.  Block inputs share
// outlier channels, so Q^, K^, V^ rows carry a large component common to all
// tokens; two exact identities cancel it (the weights of a softmax row sum to
// one, a row of dS sums to zero) and the kernels keep both under rounding: O
// is divided by the sum of the bf16 weights that entered its product, and dS
// enters the dQ and dK products as a hi + lo pair of bf16 terms.  The online
// maximum is kept integral (a power-of-two rescaling is exact), so the bf16
// weights of a row are bf16(2^(t - ceil(max t))) up to one common power of
// two, independent of the order of the key tiles.
#include <math.h>

#include "common.h"
#include "oq_internal.h"

namespace oq {
namespace {

constexpr int AT = 64;          // queries / keys per tile
constexpr int ANT = 256;        // threads per workgroup (4 waves)
constexpr int TP = 72;          // bf16 pitch of a transposed [d][64] or [16][64] LDS row (144 B)

typedef uint16_t bf16raw;

OQ_DEV bf16x8_t bits_as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }
OQ_DEV f32x4_t mfma(bf16x8_t a, bf16x8_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
OQ_DEV uint32_t pack2(float a, float b) { return f2bf2(a, b); }

// Row-major [64][DH] bf16 tile, 16-byte chunk c of row r at slot c ^ (r & (NCH-1)).
template <int DH>
OQ_DEV void load_tile_rm(uint4* lds, const bf16raw* g, int64_t ld, int tid) {
  constexpr int NCH = DH / 8;
#pragma unroll
  for (int i = 0; i < AT * NCH / ANT; ++i) {
    const int idx = tid + ANT * i;
    const int r = idx / NCH, c = idx % NCH;
    lds[r * NCH + (c ^ (r & (NCH - 1)))] = *reinterpret_cast<const uint4*>(g + r * ld + 8 * c);
  }
}
template <int DH>
OQ_DEV bf16x8_t read_rm(const uint4* lds, int r, int c) {
  constexpr int NCH = DH / 8;
  return bits_as_bf16x8(lds[r * NCH + (c ^ (r & (NCH - 1)))]);
}
// Transposed [DH][64] bf16 tile with row pitch TP (the 64 tile rows become columns).
template <int DH>
OQ_DEV void load_tile_tr(bf16raw* lds, const bf16raw* g, int64_t ld, int tid) {
  constexpr int NCH = DH / 8;
#pragma unroll
  for (int i = 0; i < AT * NCH / ANT; ++i) {
    const int idx = tid + ANT * i;
    const int r = idx % AT, c = idx / AT;        // consecutive lanes: consecutive rows
    const uint4 v = *reinterpret_cast<const uint4*>(g + r * ld + 8 * c);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      lds[(8 * c + 2 * e) * TP + r] = bf16raw(w[e] & 0xffffu);
      lds[(8 * c + 2 * e + 1) * TP + r] = bf16raw(w[e] >> 16);
    }
  }
}
// 8 consecutive bf16 of row `row` at column `col` (a multiple of 8) of a
// pitch-TP tile.
OQ_DEV bf16x8_t read_tr8(const bf16raw* lds, int row, int col) {
  return bits_as_bf16x8(*reinterpret_cast<const uint4*>(lds + row * TP + col));
}
// columns col .. col+3 and col+16 .. col+19 of row `row` (the permuted
// k-order that matches a C-layout operand, see the forward)
OQ_DEV bf16x8_t read_tr_perm(const bf16raw* lds, int row, int col) {
  const uint2 a = *reinterpret_cast<const uint2*>(lds + row * TP + col);
  const uint2 b = *reinterpret_cast<const uint2*>(lds + row * TP + col + 16);
  return bits_as_bf16x8(make_uint4(a.x, a.y, b.x, b.y));
}

// ------------------------------------------------------------------ forward
template <int DH>
__global__ __launch_bounds__(ANT) void attn_fwd_kernel(const bf16raw* __restrict__ Q,
                                                       const bf16raw* __restrict__ K,
                                                       const bf16raw* __restrict__ V, int S,
                                                       int H, int Hkv, float* __restrict__ O,
                                                       float* __restrict__ LSE, int64_t T) {
  constexpr int KS = DH / 32;        // k-steps of the S product
  constexpr int JD = DH / 16;        // 16-row tiles of O^T
  __shared__ uint4 sK[AT * DH / 8];
  __shared__ __attribute__((aligned(16))) bf16raw sVt[DH * TP];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int fr = lane & 15, fk = lane >> 4;
  const int ntile = S / AT;
  const int qt = ntile - 1 - int(blockIdx.x);          // longest tiles first
  const int h = blockIdx.y, b = blockIdx.z;
  const int g = h / (H / Hkv);
  const int64_t ldq = int64_t(H) * DH, ldk = int64_t(Hkv) * DH;
  const int64_t row0 = int64_t(b) * S;
  const int qrow = qt * AT + 16 * wave + fr;            // this lane's query within the sample
  const float sc = 1.4426950408889634f / sqrtf(float(DH));

  bf16x8_t qf[KS];
  {
    const bf16raw* qp = Q + (row0 + qrow) * ldq + int64_t(h) * DH;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[ks] = bits_as_bf16x8(*reinterpret_cast<const uint4*>(qp + 32 * ks + 8 * fk));
  }
  f32x4_t acc[JD];
#pragma unroll
  for (int j = 0; j < JD; ++j) acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, l = 0.f, l_b = 0.f;

  for (int kt = 0; kt <= qt; ++kt) {
    __syncthreads();
    const int64_t krow = row0 + int64_t(kt) * AT;
    load_tile_rm<DH>(sK, K + krow * ldk + int64_t(g) * DH, ldk, tid);
    load_tile_tr<DH>(sVt, V + krow * ldk + int64_t(g) * DH, ldk, tid);
    __syncthreads();
    // S^T [64 keys x 16 queries of this wave]
    f32x4_t st[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      st[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        st[i] = mfma(read_rm<DH>(sK, 16 * i + fr, 4 * ks + fk), qf[ks], st[i]);
    }
    float mt = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = kt * AT + 16 * i + 4 * fk + r;
        float t = st[i][r] * sc;
        if (key > qrow) t = -INFINITY;
        st[i][r] = t;
        mt = fmaxf(mt, t);
      }
    mt = fmaxf(mt, __shfl_xor(mt, 16));
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    // the running maximum stays an integer, so every rescaling below is an
    // exact power of two: each weight that reaches the PV product equals
    // bf16(2^(t - M)) times a power of two, M the row's final maximum,
    // whatever the tile order
    const float mn = fmaxf(m, ceilf(mt));
    const float alpha = m == -INFINITY ? 0.0f : ldexpf(1.0f, int(m - mn));
    float ls = 0.f;
    bf16x8_t pb[2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = exp2f(st[i][r] - mn);
        st[i][r] = p;
        ls += p;
      }
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2)
      pb[k2] = bits_as_bf16x8(make_uint4(pack2(st[2 * k2][0], st[2 * k2][1]),
                                         pack2(st[2 * k2][2], st[2 * k2][3]),
                                         pack2(st[2 * k2 + 1][0], st[2 * k2 + 1][1]),
                                         pack2(st[2 * k2 + 1][2], st[2 * k2 + 1][3])));
    // the weights the PV product sees are the bf16 values: their own sum
    // normalises O, so O stays an exact weighted mean of V rows (a component
    // shared by every V row passes through unchanged); l (unrounded) gives LSE
    float lr = 0.f;
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      const uint4 u = __builtin_bit_cast(uint4, pb[k2]);
      const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int e = 0; e < 4; ++e)
        lr += __uint_as_float(w4[e] << 16) + __uint_as_float(w4[e] & 0xffff0000u);
    }
    ls += __shfl_xor(ls, 16);
    ls += __shfl_xor(ls, 32);
    lr += __shfl_xor(lr, 16);
    lr += __shfl_xor(lr, 32);
    l = l * alpha + ls;
    l_b = l_b * alpha + lr;
    m = mn;
#pragma unroll
    for (int j = 0; j < JD; ++j) {
      acc[j] = acc[j] * alpha;
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2)
        acc[j] = mfma(read_tr_perm(sVt, 16 * j + fr, 32 * k2 + 4 * fk), pb[k2], acc[j]);
    }
  }
  const float inv = 1.0f / l_b;
  float* op = O + (row0 + qrow) * ldq + int64_t(h) * DH;
#pragma unroll
  for (int j = 0; j < JD; ++j)
    *reinterpret_cast<float4*>(op + 16 * j + 4 * fk) =
        make_float4(acc[j][0] * inv, acc[j][1] * inv, acc[j][2] * inv, acc[j][3] * inv);
  if (fk == 0) LSE[int64_t(h) * T + row0 + qrow] = m + log2f(l);
}

// ------------------------------------------------------------------ backward: dK, dV
template <int DH>
__global__ __launch_bounds__(ANT) void attn_bwd_dkv_kernel(
    const bf16raw* __restrict__ Q, const bf16raw* __restrict__ K, const bf16raw* __restrict__ V,
    const bf16raw* __restrict__ dO, const float* __restrict__ LSE, const float* __restrict__ Dl,
    int S, int H, int Hkv, int64_t T, float* __restrict__ dK, float* __restrict__ dV) {
  constexpr int KS = DH / 32, JD = DH / 16;
  __shared__ uint4 sQ[AT * DH / 8];
  __shared__ uint4 sdO[AT * DH / 8];
  __shared__ __attribute__((aligned(16))) bf16raw sQt[DH * TP];
  __shared__ __attribute__((aligned(16))) bf16raw sdOt[DH * TP];
  __shared__ __attribute__((aligned(16))) bf16raw sP[4][16 * TP];
  __shared__ __attribute__((aligned(16))) bf16raw sPl[4][16 * TP];
  __shared__ float sL[AT], sD[AT];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int fr = lane & 15, fk = lane >> 4;
  const int ntile = S / AT;
  const int kt = int(blockIdx.x), g = blockIdx.y, b = blockIdx.z;
  const int grp = H / Hkv;
  const int64_t ldq = int64_t(H) * DH, ldk = int64_t(Hkv) * DH;
  const int64_t row0 = int64_t(b) * S;
  const int key_w = kt * AT + 16 * wave;                // this wave's first key
  const float sc = 1.4426950408889634f / sqrtf(float(DH));
  const float rs = 1.0f / sqrtf(float(DH));

  bf16x8_t kf[KS], vf[KS];
  {
    const bf16raw* kp = K + (row0 + key_w + fr) * ldk + int64_t(g) * DH;
    const bf16raw* vp = V + (row0 + key_w + fr) * ldk + int64_t(g) * DH;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      kf[ks] = bits_as_bf16x8(*reinterpret_cast<const uint4*>(kp + 32 * ks + 8 * fk));
      vf[ks] = bits_as_bf16x8(*reinterpret_cast<const uint4*>(vp + 32 * ks + 8 * fk));
    }
  }
  f32x4_t adk[JD], adv[JD];
#pragma unroll
  for (int j = 0; j < JD; ++j) adk[j] = adv[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  for (int hq = g * grp; hq < (g + 1) * grp; ++hq) {
    for (int qt = kt; qt < ntile; ++qt) {
      __syncthreads();
      const int64_t qrow0 = row0 + int64_t(qt) * AT;
      load_tile_rm<DH>(sQ, Q + qrow0 * ldq + int64_t(hq) * DH, ldq, tid);
      load_tile_rm<DH>(sdO, dO + qrow0 * ldq + int64_t(hq) * DH, ldq, tid);
      load_tile_tr<DH>(sQt, Q + qrow0 * ldq + int64_t(hq) * DH, ldq, tid);
      load_tile_tr<DH>(sdOt, dO + qrow0 * ldq + int64_t(hq) * DH, ldq, tid);
      if (tid < AT) {
        sL[tid] = LSE[int64_t(hq) * T + qrow0 + tid];
        sD[tid] = Dl[int64_t(hq) * T + qrow0 + tid];
      }
      __syncthreads();
      // S^T and dP^T [16 keys x 64 queries]: lane holds key 4 fk + r, query 16 jn + fr
      f32x4_t st[4], dp[4];
#pragma unroll
      for (int jn = 0; jn < 4; ++jn) {
        st[jn] = dp[jn] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          st[jn] = mfma(kf[ks], read_rm<DH>(sQ, 16 * jn + fr, 4 * ks + fk), st[jn]);
          dp[jn] = mfma(vf[ks], read_rm<DH>(sdO, 16 * jn + fr, 4 * ks + fk), dp[jn]);
        }
      }
      bf16raw* pw = sP[wave];
      // P^T into this wave's LDS rows; then dS^T into the same rows (after dV)
#pragma unroll
      for (int jn = 0; jn < 4; ++jn) {
        const int ql = 16 * jn + fr;
        const int q = qt * AT + ql;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = key_w + 4 * fk + r;
          float p = key > q ? 0.0f : exp2f(st[jn][r] * sc - sL[ql]);
          st[jn][r] = p;
          dp[jn][r] = p * (dp[jn][r] - sD[ql]) * rs;     // dS^T (with the 1/sqrt(d) of the logits)
          pw[(4 * fk + r) * TP + ql] = f2bf(p);
        }
      }
      // dV += P^T dO: A = P^T rows (keys), B = dO^T rows (d); k = queries
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        const bf16x8_t a = read_tr8(pw, fr, 32 * k2 + 8 * fk);
#pragma unroll
        for (int j = 0; j < JD; ++j) adv[j] = mfma(a, read_tr8(sdOt, 16 * j + fr, 32 * k2 + 8 * fk), adv[j]);
      }
      // dK += dS^T Q with dS split into two bf16 terms (hi + lo, 16 significant
      // bits): a component shared by all queries' Q rows would otherwise meet
      // the rounding of dS unreduced.  The wave rewrites only its own rows,
      // after its own reads of them.
      bf16raw* pwl = sPl[wave];
#pragma unroll
      for (int jn = 0; jn < 4; ++jn)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const bf16raw hi = f2bf(dp[jn][r]);
          pw[(4 * fk + r) * TP + 16 * jn + fr] = hi;
          pwl[(4 * fk + r) * TP + 16 * jn + fr] = f2bf(dp[jn][r] - bf2f(hi));
        }
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        const bf16x8_t a = read_tr8(pw, fr, 32 * k2 + 8 * fk);
        const bf16x8_t al = read_tr8(pwl, fr, 32 * k2 + 8 * fk);
#pragma unroll
        for (int j = 0; j < JD; ++j) {
          const bf16x8_t bq = read_tr8(sQt, 16 * j + fr, 32 * k2 + 8 * fk);
          adk[j] = mfma(al, bq, mfma(a, bq, adk[j]));
        }
      }
    }
  }
  // lane holds dK/dV[key_w + 4 fk + r][16 j + fr]
#pragma unroll
  for (int j = 0; j < JD; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t o = (row0 + key_w + 4 * fk + r) * ldk + int64_t(g) * DH + 16 * j + fr;
      dK[o] = adk[j][r];
      dV[o] = adv[j][r];
    }
}

// ------------------------------------------------------------------ backward: dQ
template <int DH>
__global__ __launch_bounds__(ANT) void attn_bwd_dq_kernel(
    const bf16raw* __restrict__ Q, const bf16raw* __restrict__ K, const bf16raw* __restrict__ V,
    const bf16raw* __restrict__ dO, const float* __restrict__ LSE, float* __restrict__ Dl,
    int S, int H, int Hkv, int64_t T, float* __restrict__ dQ) {
  constexpr int KS = DH / 32, JD = DH / 16;
  __shared__ uint4 sK[AT * DH / 8];
  __shared__ uint4 sV[AT * DH / 8];
  __shared__ __attribute__((aligned(16))) bf16raw sKt[DH * TP];
  __shared__ __attribute__((aligned(16))) bf16raw sS[4][16 * TP];
  __shared__ __attribute__((aligned(16))) bf16raw sSl[4][16 * TP];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int fr = lane & 15, fk = lane >> 4;
  const int ntile = S / AT;
  const int qt = ntile - 1 - int(blockIdx.x);
  const int h = blockIdx.y, b = blockIdx.z;
  const int g = h / (H / Hkv);
  const int64_t ldq = int64_t(H) * DH, ldk = int64_t(Hkv) * DH;
  const int64_t row0 = int64_t(b) * S;
  const int q_w = qt * AT + 16 * wave;                  // this wave's first query
  const float sc = 1.4426950408889634f / sqrtf(float(DH));
  const float rs = 1.0f / sqrtf(float(DH));

  bf16x8_t qf[KS], df[KS];
  {
    const bf16raw* qp = Q + (row0 + q_w + fr) * ldq + int64_t(h) * DH;
    const bf16raw* dp = dO + (row0 + q_w + fr) * ldq + int64_t(h) * DH;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      qf[ks] = bits_as_bf16x8(*reinterpret_cast<const uint4*>(qp + 32 * ks + 8 * fk));
      df[ks] = bits_as_bf16x8(*reinterpret_cast<const uint4*>(dp + 32 * ks + 8 * fk));
    }
  }
  // the rows this lane's accumulators hold: queries q_w + 4 fk + r
  float lse[4], dl[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    lse[r] = LSE[int64_t(h) * T + row0 + q_w + 4 * fk + r];
    dl[r] = 0.f;
  }
  // sweep 1: D = sum_j P_ij dP_ij from the very probabilities the gradients
  // use, so that every row of dS sums to zero to fp32 rounding
  for (int kt = 0; kt <= qt; ++kt) {
    __syncthreads();
    const int64_t krow = row0 + int64_t(kt) * AT;
    load_tile_rm<DH>(sK, K + krow * ldk + int64_t(g) * DH, ldk, tid);
    load_tile_rm<DH>(sV, V + krow * ldk + int64_t(g) * DH, ldk, tid);
    __syncthreads();
#pragma unroll
    for (int jn = 0; jn < 4; ++jn) {
      f32x4_t st = f32x4_t{0.f, 0.f, 0.f, 0.f}, dp = st;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        st = mfma(qf[ks], read_rm<DH>(sK, 16 * jn + fr, 4 * ks + fk), st);
        dp = mfma(df[ks], read_rm<DH>(sV, 16 * jn + fr, 4 * ks + fk), dp);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = kt * AT + 16 * jn + fr;
        if (key <= q_w + 4 * fk + r) dl[r] += exp2f(st[r] * sc - lse[r]) * dp[r];
      }
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) dl[r] += __shfl_xor(dl[r], o);
  }
  if (fr == 0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) Dl[int64_t(h) * T + row0 + q_w + 4 * fk + r] = dl[r];
  }
  f32x4_t adq[JD];
#pragma unroll
  for (int j = 0; j < JD; ++j) adq[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  for (int kt = 0; kt <= qt; ++kt) {
    __syncthreads();
    const int64_t krow = row0 + int64_t(kt) * AT;
    load_tile_rm<DH>(sK, K + krow * ldk + int64_t(g) * DH, ldk, tid);
    load_tile_rm<DH>(sV, V + krow * ldk + int64_t(g) * DH, ldk, tid);
    load_tile_tr<DH>(sKt, K + krow * ldk + int64_t(g) * DH, ldk, tid);
    __syncthreads();
    // S and dP [16 queries x 64 keys]: lane holds query 4 fk + r, key 16 jn + fr
    f32x4_t st[4], dp[4];
#pragma unroll
    for (int jn = 0; jn < 4; ++jn) {
      st[jn] = dp[jn] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        st[jn] = mfma(qf[ks], read_rm<DH>(sK, 16 * jn + fr, 4 * ks + fk), st[jn]);
        dp[jn] = mfma(df[ks], read_rm<DH>(sV, 16 * jn + fr, 4 * ks + fk), dp[jn]);
      }
    }
    bf16raw* sw = sS[wave];
#pragma unroll
    for (int jn = 0; jn < 4; ++jn)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int q = q_w + 4 * fk + r;
        const int key = kt * AT + 16 * jn + fr;
        const float p = key > q ? 0.0f : exp2f(st[jn][r] * sc - lse[r]);
        dp[jn][r] = p * (dp[jn][r] - dl[r]) * rs;
      }
    // dQ += dS K: A = dS rows (queries), B = K^T rows (d); k = keys.  dS as
    // hi + lo bf16 terms: each row of dS sums to zero, so a component shared
    // by all K rows cancels in the exact product and must not survive the
    // rounding of dS.  Wave-private rows, rewritten after their reads.
    bf16raw* swl = sSl[wave];
#pragma unroll
    for (int jn = 0; jn < 4; ++jn)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bf16raw hi = f2bf(dp[jn][r]);
        sw[(4 * fk + r) * TP + 16 * jn + fr] = hi;
        swl[(4 * fk + r) * TP + 16 * jn + fr] = f2bf(dp[jn][r] - bf2f(hi));
      }
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      const bf16x8_t a = read_tr8(sw, fr, 32 * k2 + 8 * fk);
      const bf16x8_t al = read_tr8(swl, fr, 32 * k2 + 8 * fk);
#pragma unroll
      for (int j = 0; j < JD; ++j) {
        const bf16x8_t bk = read_tr8(sKt, 16 * j + fr, 32 * k2 + 8 * fk);
        adq[j] = mfma(al, bk, mfma(a, bk, adq[j]));
      }
    }
  }
#pragma unroll
  for (int j = 0; j < JD; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      dQ[(row0 + q_w + 4 * fk + r) * ldq + int64_t(h) * DH + 16 * j + fr] = adq[j][r];
}

template <int DH>
hipError_t attn_fwd_t(const void* Q, const void* K, const void* V, int64_t T, int S, int H,
                      int Hkv, float* O, float* LSE, hipStream_t st) {
  const dim3 grid(unsigned(S / AT), unsigned(H), unsigned(T / S));
  hipLaunchKernelGGL(attn_fwd_kernel<DH>, grid, dim3(ANT), 0, st, static_cast<const bf16raw*>(Q),
                     static_cast<const bf16raw*>(K), static_cast<const bf16raw*>(V), S, H, Hkv, O,
                     LSE, T);
  return hipGetLastError();
}

template <int DH>
hipError_t attn_bwd_t(const void* Q, const void* K, const void* V, const void* dO,
                      const float* LSE, int64_t T, int S, int H, int Hkv, float* Dl, float* dQ,
                      float* dK, float* dV, hipStream_t st) {
  // dQ first: it also writes D, which the dK/dV kernel reads
  hipLaunchKernelGGL(attn_bwd_dq_kernel<DH>, dim3(unsigned(S / AT), unsigned(H), unsigned(T / S)),
                     dim3(ANT), 0, st, static_cast<const bf16raw*>(Q), static_cast<const bf16raw*>(K),
                     static_cast<const bf16raw*>(V), static_cast<const bf16raw*>(dO), LSE, Dl, S, H,
                     Hkv, T, dQ);
  hipLaunchKernelGGL(attn_bwd_dkv_kernel<DH>, dim3(unsigned(S / AT), unsigned(Hkv), unsigned(T / S)),
                     dim3(ANT), 0, st, static_cast<const bf16raw*>(Q), static_cast<const bf16raw*>(K),
                     static_cast<const bf16raw*>(V), static_cast<const bf16raw*>(dO), LSE, Dl, S, H,
                     Hkv, T, dK, dV);
  return hipGetLastError();
}

}  // namespace

bool attn_supported(int64_t T, int S, int H, int Hkv, int dh) {
  return (dh == 64 || dh == 128) && S > 0 && S % AT == 0 && T > 0 && T % S == 0 && H > 0 &&
         Hkv > 0 && H % Hkv == 0 && T / S <= 65535 && H <= 65535;
}

hipError_t attn_fwd(const void* Q, const void* K, const void* V, int64_t T, int S, int H, int Hkv,
                    int dh, float* O, float* LSE, hipStream_t st) {
  if (!attn_supported(T, S, H, Hkv, dh)) return hipErrorInvalidValue;
  return dh == 128 ? attn_fwd_t<128>(Q, K, V, T, S, H, Hkv, O, LSE, st)
                   : attn_fwd_t<64>(Q, K, V, T, S, H, Hkv, O, LSE, st);
}

hipError_t attn_bwd(const void* Q, const void* K, const void* V, const void* dO, const float* LSE,
                    int64_t T, int S, int H, int Hkv, int dh, float* Dl, float* dQ, float* dK,
                    float* dV, hipStream_t st) {
  if (!attn_supported(T, S, H, Hkv, dh)) return hipErrorInvalidValue;
  return dh == 128 ? attn_bwd_t<128>(Q, K, V, dO, LSE, T, S, H, Hkv, Dl, dQ, dK, dV, st)
                   : attn_bwd_t<64>(Q, K, V, dO, LSE, T, S, H, Hkv, Dl, dQ, dK, dV, st);
}

}  // namespace oq
