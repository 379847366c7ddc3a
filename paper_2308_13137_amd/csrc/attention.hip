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

typedef uint16_t bf16raw;

OQ_DEV bf16x8_t bits_as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }
OQ_DEV f32x4_t mfma(bf16x8_t a, bf16x8_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
OQ_DEV uint32_t pack2(float a, float b) { return f2bf2(a, b); }

// Row-major [64][DH] bf16 tile ("K layout"), 16-byte chunk c of row r at
// slot c ^ (r & (NCH-1)).
template <int DH>
OQ_DEV bf16x8_t read_rm(const uint4* lds, int r, int c) {
  constexpr int NCH = DH / 8;
  return bits_as_bf16x8(lds[r * NCH + (c ^ (r & (NCH - 1)))]);
}

// ------------------------------------------------------------------ forward
// Row-major [64][DH] bf16 tile in 32-byte blocks, block b of row r at
// b ^ vswz(r): the four rows one transposed read of a 16-lane group touches
// (and the next group's four) fall in distinct banks.
template <int DH>
OQ_DEV int vswz(int r) {
  return (r + 4 * (r >> 3)) & (DH / 16 - 1);
}
// Global -> registers: this thread's chunks of a 64-row tile (NCH 16-byte
// chunks per row), chunk idx = tid + ANT * i.
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
template <int DH>
OQ_DEV void tile_to_regs(u32x4_t (&v)[AT * DH / 8 / ANT], const bf16raw* g, int64_t ld, int tid) {
  constexpr int NCH = DH / 8;
#pragma unroll
  for (int i = 0; i < AT * NCH / ANT; ++i) {
    const int idx = tid + ANT * i;
    v[i] = *reinterpret_cast<const u32x4_t*>(g + (idx / NCH) * ld + 8 * (idx % NCH));
  }
}
// registers -> LDS, K layout (16-byte chunk c of row r at c ^ (r & (NCH-1)))
template <int DH>
OQ_DEV void regs_to_k(uint4* lds, const u32x4_t (&v)[AT * DH / 8 / ANT], int tid) {
  constexpr int NCH = DH / 8;
#pragma unroll
  for (int i = 0; i < AT * NCH / ANT; ++i) {
    const int idx = tid + ANT * i;
    const int r = idx / NCH, c = idx % NCH;
    reinterpret_cast<u32x4_t*>(lds)[r * NCH + (c ^ (r & (NCH - 1)))] = v[i];
  }
}
// registers -> LDS, V layout (32-byte block b of row r at b ^ vswz(r))
template <int DH>
OQ_DEV void regs_to_v(uint4* lds, const u32x4_t (&v)[AT * DH / 8 / ANT], int tid) {
  constexpr int NCH = DH / 8;
#pragma unroll
  for (int i = 0; i < AT * NCH / ANT; ++i) {
    const int idx = tid + ANT * i;
    const int r = idx / NCH, c = idx % NCH;
    reinterpret_cast<u32x4_t*>(lds)[r * NCH + 2 * ((c >> 1) ^ vswz<DH>(r)) + (c & 1)] = v[i];
  }
}
// A operand of O^T = V^T P for rows d = 16 j .. 16 j + 15 and the k-chunk k2,
// in the k order of the P operand: lane (fk, i) needs keys 32 k2 + 4 fk + 0..3
// and 32 k2 + 16 + 4 fk + 0..3 of column d = 16 j + i.  ds_read_b64_tr_b16
// gives lane i of a 16-lane group four consecutive rows k0..k0+3 of column
// 16 j + i when lane j' of the group points at row k0 + j'/4, columns
// 16 j + 4 (j' % 4) .. + 3.
template <int DH>
OQ_DEV bf16x8_t v_frag(const uint4* sV, int j, int k2, int lane) {
  typedef short v4i16 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) v4i16 lds_v4;
  const int fk = lane >> 4, jj = lane & 15;
  const int r0 = 32 * k2 + 4 * fk + (jj >> 2), r1 = r0 + 16;
  const char* base = reinterpret_cast<const char*>(sV);
  const char* a0 = base + r0 * (2 * DH) + 32 * (j ^ vswz<DH>(r0)) + 8 * (jj & 3);
  const char* a1 = base + r1 * (2 * DH) + 32 * (j ^ vswz<DH>(r1)) + 8 * (jj & 3);
  const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4*)(a0));
  const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4*)(a1));
  return __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

template <int DH>
__global__ __launch_bounds__(ANT) void attn_fwd_kernel(const bf16raw* __restrict__ Q,
                                                       const bf16raw* __restrict__ K,
                                                       const bf16raw* __restrict__ V, int S,
                                                       int H, int Hkv, float* __restrict__ O,
                                                       float* __restrict__ LSE, int64_t T) {
  constexpr int KS = DH / 32;        // k-steps of the S product
  constexpr int JD = DH / 16;        // 16-row tiles of O^T
  constexpr int NR = AT * DH / 8 / ANT;
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  __shared__ uint4 sK[AT * DH / 8];
  __shared__ uint4 sV[AT * DH / 8];
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
  const bf16x2_t ones = {(__bf16)1.0f, (__bf16)1.0f};

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
  u32x4_t kr[NR], vr[NR];
  tile_to_regs<DH>(kr, K + row0 * ldk + int64_t(g) * DH, ldk, tid);
  tile_to_regs<DH>(vr, V + row0 * ldk + int64_t(g) * DH, ldk, tid);

  for (int kt = 0; kt <= qt; ++kt) {
    __syncthreads();
    regs_to_k<DH>(sK, kr, tid);
    regs_to_v<DH>(sV, vr, tid);
    __syncthreads();
    {                                                    // the next tile, in flight meanwhile
      const int64_t krow = row0 + int64_t(kt < qt ? kt + 1 : kt) * AT;
      tile_to_regs<DH>(kr, K + krow * ldk + int64_t(g) * DH, ldk, tid);
      tile_to_regs<DH>(vr, V + krow * ldk + int64_t(g) * DH, ldk, tid);
    }
    // S^T [64 keys x 16 queries of this wave]: lane holds key 16 i + 4 fk + r, query fr
    f32x4_t st[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      st[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        st[i] = mfma(read_rm<DH>(sK, 16 * i + fr, 4 * ks + fk), qf[ks], st[i]);
    }
    if (kt == qt) {                                      // the diagonal tile: causal mask
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (kt * AT + 16 * i + 4 * fk + r > qrow) st[i][r] = -INFINITY;
    }
    float mt = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) mt = fmaxf(fmaxf(mt, fmaxf(st[i][0], st[i][1])), fmaxf(st[i][2], st[i][3]));
    mt = fmaxf(mt, __shfl_xor(mt, 16));
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    // the running maximum stays an integer, so every rescaling is an exact
    // power of two: each weight reaching the PV product is bf16(2^(t - M))
    // times a power of two, M the row's final maximum, whatever the tile order
    const float mn = fmaxf(m, ceilf(mt * sc));
    float ls = 0.f, lr = 0.f;
    bf16x8_t pb[2];
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = 2 * k2 + (e >> 1), r0 = 2 * (e & 1);
        const float p0 = __builtin_amdgcn_exp2f(fmaf(st[i][r0], sc, -mn));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(st[i][r0 + 1], sc, -mn));
        ls += p0 + p1;
        w[e] = pack2(p0, p1);
        // the weights the PV product sees are these bf16 values: their own
        // sum normalises O (an exact weighted mean of V rows); l (unrounded)
        // gives LSE
        lr = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w[e]), ones, lr, false);
      }
      pb[k2] = bits_as_bf16x8(make_uint4(w[0], w[1], w[2], w[3]));
    }
    ls += __shfl_xor(ls, 16);
    ls += __shfl_xor(ls, 32);
    lr += __shfl_xor(lr, 16);
    lr += __shfl_xor(lr, 32);
    if (__any(mn != m)) {
      const float alpha = m == -INFINITY ? 0.0f : ldexpf(1.0f, int(m - mn));
      l *= alpha;
      l_b *= alpha;
#pragma unroll
      for (int j = 0; j < JD; ++j) acc[j] = acc[j] * alpha;
    }
    l += ls;
    l_b += lr;
    m = mn;
#pragma unroll
    for (int j = 0; j < JD; ++j)
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) acc[j] = mfma(v_frag<DH>(sV, j, k2, lane), pb[k2], acc[j]);
  }
  const float inv = 1.0f / l_b;
  float* op = O + (row0 + qrow) * ldq + int64_t(h) * DH;
#pragma unroll
  for (int j = 0; j < JD; ++j)
    *reinterpret_cast<float4*>(op + 16 * j + 4 * fk) =
        make_float4(acc[j][0] * inv, acc[j][1] * inv, acc[j][2] * inv, acc[j][3] * inv);
  if (fk == 0) LSE[int64_t(h) * T + row0 + qrow] = m + log2f(l);
}

// The same forward with 32 queries per wave (128 per workgroup, S a multiple
// of 128): every K and V fragment read from LDS feeds two matrix
// instructions, one per 16-query half, which halves the LDS traffic per
// instruction.  Arithmetic per query is the kernel's above, unchanged.
template <int DH>
__global__ __launch_bounds__(ANT) void attn_fwd2_kernel(const bf16raw* __restrict__ Q,
                                                        const bf16raw* __restrict__ K,
                                                        const bf16raw* __restrict__ V, int S,
                                                        int H, int Hkv, float* __restrict__ O,
                                                        float* __restrict__ LSE, int64_t T) {
  constexpr int KS = DH / 32;
  constexpr int JD = DH / 16;
  constexpr int NR = AT * DH / 8 / ANT;
  constexpr int QW = 2 * AT;                           // queries per workgroup
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  __shared__ uint4 sK[AT * DH / 8];
  __shared__ uint4 sV[AT * DH / 8];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int fr = lane & 15, fk = lane >> 4;
  const int nq = S / QW;
  const int qt = nq - 1 - int(blockIdx.x);             // longest tiles first
  const int h = blockIdx.y, b = blockIdx.z;
  const int g = h / (H / Hkv);
  const int64_t ldq = int64_t(H) * DH, ldk = int64_t(Hkv) * DH;
  const int64_t row0 = int64_t(b) * S;
  int qrow[2];
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) qrow[hh] = qt * QW + 32 * wave + 16 * hh + fr;
  const float sc = 1.4426950408889634f / sqrtf(float(DH));
  const bf16x2_t ones = {(__bf16)1.0f, (__bf16)1.0f};

  bf16x8_t qf[2][KS];
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const bf16raw* qp = Q + (row0 + qrow[hh]) * ldq + int64_t(h) * DH;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[hh][ks] = bits_as_bf16x8(*reinterpret_cast<const uint4*>(qp + 32 * ks + 8 * fk));
  }
  f32x4_t acc[2][JD];
#pragma unroll
  for (int hh = 0; hh < 2; ++hh)
#pragma unroll
    for (int j = 0; j < JD; ++j) acc[hh][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m[2] = {-INFINITY, -INFINITY}, l[2] = {0.f, 0.f}, l_b[2] = {0.f, 0.f};
  u32x4_t kr[NR], vr[NR];
  tile_to_regs<DH>(kr, K + row0 * ldk + int64_t(g) * DH, ldk, tid);
  tile_to_regs<DH>(vr, V + row0 * ldk + int64_t(g) * DH, ldk, tid);
  const int nk = 2 * qt + 2;                           // key tiles up to the diagonal
  for (int kt = 0; kt < nk; ++kt) {
    __syncthreads();
    regs_to_k<DH>(sK, kr, tid);
    regs_to_v<DH>(sV, vr, tid);
    __syncthreads();
    {
      const int64_t krow = row0 + int64_t(kt + 1 < nk ? kt + 1 : kt) * AT;
      tile_to_regs<DH>(kr, K + krow * ldk + int64_t(g) * DH, ldk, tid);
      tile_to_regs<DH>(vr, V + krow * ldk + int64_t(g) * DH, ldk, tid);
    }
    // S^T [64 keys x 16 queries] per half: lane holds key 16 i + 4 fk + r, query fr
    f32x4_t st[2][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      st[0][i] = st[1][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8_t kf = read_rm<DH>(sK, 16 * i + fr, 4 * ks + fk);
        st[0][i] = mfma(kf, qf[0][ks], st[0][i]);
        st[1][i] = mfma(kf, qf[1][ks], st[1][i]);
      }
    }
    if (kt >= 2 * qt) {                                // the tiles the diagonal crosses
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (kt * AT + 16 * i + 4 * fk + r > qrow[hh]) st[hh][i][r] = -INFINITY;
    }
    bf16x8_t pb[2][2];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      float mt = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        mt = fmaxf(fmaxf(mt, fmaxf(st[hh][i][0], st[hh][i][1])), fmaxf(st[hh][i][2], st[hh][i][3]));
      mt = fmaxf(mt, __shfl_xor(mt, 16));
      mt = fmaxf(mt, __shfl_xor(mt, 32));
      const float mn = fmaxf(m[hh], ceilf(mt * sc));
      float ls = 0.f, lr = 0.f;
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        uint32_t w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i = 2 * k2 + (e >> 1), r0 = 2 * (e & 1);
          const float p0 = __builtin_amdgcn_exp2f(fmaf(st[hh][i][r0], sc, -mn));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(st[hh][i][r0 + 1], sc, -mn));
          ls += p0 + p1;
          w[e] = pack2(p0, p1);
          lr = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w[e]), ones, lr, false);
        }
        pb[hh][k2] = bits_as_bf16x8(make_uint4(w[0], w[1], w[2], w[3]));
      }
      ls += __shfl_xor(ls, 16);
      ls += __shfl_xor(ls, 32);
      lr += __shfl_xor(lr, 16);
      lr += __shfl_xor(lr, 32);
      if (__any(mn != m[hh])) {
        // a row whose first tile is wholly masked keeps m = -inf until its
        // first key arrives: alpha 0 leaves its (zero) sums as they are
        const float alpha = m[hh] == -INFINITY ? 0.0f : ldexpf(1.0f, int(m[hh] - mn));
        l[hh] *= alpha;
        l_b[hh] *= alpha;
#pragma unroll
        for (int j = 0; j < JD; ++j) acc[hh][j] = acc[hh][j] * alpha;
      }
      l[hh] += ls;
      l_b[hh] += lr;
      m[hh] = mn;
    }
#pragma unroll
    for (int j = 0; j < JD; ++j)
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        const bf16x8_t vf = v_frag<DH>(sV, j, k2, lane);
        acc[0][j] = mfma(vf, pb[0][k2], acc[0][j]);
        acc[1][j] = mfma(vf, pb[1][k2], acc[1][j]);
      }
  }
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const float inv = 1.0f / l_b[hh];
    float* op = O + (row0 + qrow[hh]) * ldq + int64_t(h) * DH;
#pragma unroll
    for (int j = 0; j < JD; ++j)
      *reinterpret_cast<float4*>(op + 16 * j + 4 * fk) =
          make_float4(acc[hh][j][0] * inv, acc[hh][j][1] * inv, acc[hh][j][2] * inv,
                      acc[hh][j][3] * inv);
    if (fk == 0) LSE[int64_t(h) * T + row0 + qrow[hh]] = m[hh] + log2f(l[hh]);
  }
}

// ------------------------------------------------------------------ forward, quantised softmax
// The ablation on softmax quantisation: every query row of probabilities
// goes through Q_a (per-row asymmetric MinMax, the activation quantiser's
// fp32 order) before the product with V.  A row's range must be known before
// any of its values is quantised, so the kernel sweeps the key tiles twice:
// the first forms LSE (integral running maximum, as the forward above) and
// the extreme logits, the second recomputes P = 2^(t - LSE), quantises it
// with the row's (max, min) and accumulates O = sum P^ V (no renormalisation:
// P^ approximates the normalised row).  Row record pstat [H, T, 4]:
// (max P, min P, lowest index holding each) -- the masked entries of a row
// are zeros, so every row but a sample's last has min 0.
template <int DH>
__global__ __launch_bounds__(ANT) void attn_fwd_q_kernel(const bf16raw* __restrict__ Q,
                                                         const bf16raw* __restrict__ K,
                                                         const bf16raw* __restrict__ V, int S,
                                                         int H, int Hkv, int p_bits,
                                                         float* __restrict__ O,
                                                         float* __restrict__ LSE,
                                                         float4* __restrict__ pstat, int64_t T) {
  constexpr int KS = DH / 32, JD = DH / 16, NR = AT * DH / 8 / ANT;
  __shared__ uint4 sK[AT * DH / 8];
  __shared__ uint4 sV[AT * DH / 8];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int fr = lane & 15, fk = lane >> 4;
  const int ntile = S / AT;
  const int qt = ntile - 1 - int(blockIdx.x);
  const int h = blockIdx.y, b = blockIdx.z;
  const int g = h / (H / Hkv);
  const int64_t ldq = int64_t(H) * DH, ldk = int64_t(Hkv) * DH;
  const int64_t row0 = int64_t(b) * S;
  const int qrow = qt * AT + 16 * wave + fr;
  const float sc = 1.4426950408889634f / sqrtf(float(DH));
  const float qmax = float((1 << p_bits) - 1);

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
  float m = -INFINITY, l = 0.f, smax = -INFINITY, smin = INFINITY, lse = 0.f;
  QParams prm{};
  float pmx = 0.f, pmn = 0.f;
  int amax = INT_MAX, amin = INT_MAX;
  u32x4_t kr[NR], vr[NR];
  const int nk = qt + 1;
  auto fetch = [&](int t) {
    const int64_t krow = row0 + int64_t(t) * AT;
    tile_to_regs<DH>(kr, K + krow * ldk + int64_t(g) * DH, ldk, tid);
    tile_to_regs<DH>(vr, V + krow * ldk + int64_t(g) * DH, ldk, tid);
  };
  fetch(0);
  for (int it = 0; it < 2 * nk; ++it) {
    const int kt = it < nk ? it : it - nk;
    __syncthreads();
    regs_to_k<DH>(sK, kr, tid);
    regs_to_v<DH>(sV, vr, tid);
    __syncthreads();
    fetch(kt + 1 < nk ? kt + 1 : 0);
    f32x4_t st[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      st[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        st[i] = mfma(read_rm<DH>(sK, 16 * i + fr, 4 * ks + fk), qf[ks], st[i]);
    }
    if (kt == qt) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (kt * AT + 16 * i + 4 * fk + r > qrow) st[i][r] = -INFINITY;
    }
    if (it < nk) {
      // sweep 1: LSE as the forward forms it, and the row's extreme logits
      float mt = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          mt = fmaxf(mt, st[i][r]);
          if (st[i][r] != -INFINITY) smin = fminf(smin, st[i][r]);
        }
      smax = fmaxf(smax, mt);
      mt = fmaxf(mt, __shfl_xor(mt, 16));
      mt = fmaxf(mt, __shfl_xor(mt, 32));
      const float mn_ = fmaxf(m, ceilf(mt * sc));
      float ls = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) ls += __builtin_amdgcn_exp2f(fmaf(st[i][r], sc, -mn_));
      ls += __shfl_xor(ls, 16);
      ls += __shfl_xor(ls, 32);
      l = (m == -INFINITY ? 0.0f : l * ldexpf(1.0f, int(m - mn_))) + ls;
      m = mn_;
      if (it == nk - 1) {
        smax = fmaxf(smax, __shfl_xor(smax, 16));
        smax = fmaxf(smax, __shfl_xor(smax, 32));
        smin = fminf(smin, __shfl_xor(smin, 16));
        smin = fminf(smin, __shfl_xor(smin, 32));
        lse = m + log2f(l);
        // the row's extreme probabilities, computed as each element's is
        pmx = __builtin_amdgcn_exp2f(fmaf(smax, sc, -lse));
        pmn = qrow < S - 1 ? 0.0f : __builtin_amdgcn_exp2f(fmaf(smin, sc, -lse));
        prm = make_qparams(pmx, pmn, 1.0f, 1.0f, qmax);
      }
      continue;
    }
    // sweep 2: P, its quantisation, and O += P^ V
    bf16x8_t pb[2];
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = 2 * k2 + (e >> 1), r0 = 2 * (e & 1);
        float pq[2];
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const float p = __builtin_amdgcn_exp2f(fmaf(st[i][r0 + c], sc, -lse));
          const int key = kt * AT + 16 * i + 4 * fk + r0 + c;
          if (p == pmx) amax = min(amax, key);
          if (p == pmn) amin = min(amin, key);
          pq[c] = dequant(quant_elem(p, prm, qmax).q, prm);
        }
        w[e] = pack2(pq[0], pq[1]);
      }
      pb[k2] = bits_as_bf16x8(make_uint4(w[0], w[1], w[2], w[3]));
    }
#pragma unroll
    for (int j = 0; j < JD; ++j)
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) acc[j] = mfma(v_frag<DH>(sV, j, k2, lane), pb[k2], acc[j]);
  }
  amax = min(amax, __shfl_xor(amax, 16));
  amax = min(amax, __shfl_xor(amax, 32));
  amin = min(amin, __shfl_xor(amin, 16));
  amin = min(amin, __shfl_xor(amin, 32));
  // a masked key past the visited tiles is the first zero if none came before
  if (amin == INT_MAX) amin = qrow + 1;
  float* op = O + (row0 + qrow) * ldq + int64_t(h) * DH;
#pragma unroll
  for (int j = 0; j < JD; ++j)
    *reinterpret_cast<float4*>(op + 16 * j + 4 * fk) =
        make_float4(acc[j][0], acc[j][1], acc[j][2], acc[j][3]);
  if (fk == 0) {
    LSE[int64_t(h) * T + row0 + qrow] = lse;
    pstat[int64_t(h) * T + row0 + qrow] =
        make_float4(pmx, pmn, __int_as_float(amax), __int_as_float(amin));
  }
}

// ------------------------------------------------------------------ backward
// Operands the backward needs transposed are read from the row-major tiles
// with ds_read_b64_tr_b16: lane i of a 16-lane group receives rows
// k0 .. k0+3 of column c0 + i when lane j of the group points at row
// k0 + j/4, columns c0 + 4 (j % 4) .. + 3.
typedef short v4i16_t __attribute__((ext_vector_type(4)));
OQ_DEV v4i16_t tr4(const void* p) {
  typedef __attribute__((address_space(3))) v4i16_t lds_v4;
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4*)(p));
}
OQ_DEV bf16x8_t join(v4i16_t lo, v4i16_t hi) {
  return __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}
// Operand fragment from a [64][DH] tile in the K layout: lane (fk, i) gets
// rows kb + 8 fk + 0..7 of column cb + i (cb a multiple of 16).
template <int DH>
OQ_DEV bf16x8_t col_frag(const uint4* tile, int kb, int cb, int lane) {
  constexpr int NCH = DH / 8;
  const int fk = lane >> 4, jj = lane & 15;
  const int cc = cb + 4 * (jj & 3);
  const int r0 = kb + 8 * fk + (jj >> 2), r1 = r0 + 4;
  const char* base = reinterpret_cast<const char*>(tile);
  const char* a0 = base + r0 * (2 * DH) + 16 * ((cc >> 3) ^ (r0 & (NCH - 1))) + 2 * (cc & 7);
  const char* a1 = base + r1 * (2 * DH) + 16 * ((cc >> 3) ^ (r1 & (NCH - 1))) + 2 * (cc & 7);
  return join(tr4(a0), tr4(a1));
}
// A wave's [64][16] bf16 staging tile (row pitch TS): a lane of the product's
// C layout writes four consecutive columns of one row in one 8-byte store;
// t16_frag gives lane (fk, i) rows kb + 8 fk + 0..7 of column i.
constexpr int TS = 20;
OQ_DEV void t16_put4(bf16raw* t, int row, int col, float a, float b, float c, float d) {
  *reinterpret_cast<uint2*>(t + row * TS + col) = make_uint2(pack2(a, b), pack2(c, d));
}
OQ_DEV bf16x8_t t16_frag(const bf16raw* t, int kb, int lane) {
  const int fk = lane >> 4, jj = lane & 15;
  const int r0 = kb + 8 * fk + (jj >> 2);
  const bf16raw* a0 = t + r0 * TS + 4 * (jj & 3);
  return join(tr4(a0), tr4(a0 + 4 * TS));
}

// dK, dV: one workgroup per 64-key tile and key head; each wave owns 16 keys
// and accumulates over every query tile and query head of its group (S^T and
// dP^T recomputed from LSE and D).  P^T and dS^T pass through the wave's
// staging tiles, query-major, to become A operands.
// QP (softmax quantisation): P^ (the quantised row) enters dV, and dP goes
// through Q_a's straight-through rule: dP = m dP^ plus the routed gradients of
// the row's max and min (from the dQ kernel's first sweep).
template <int DH, bool QP>
__global__ __launch_bounds__(ANT, 2) void attn_bwd_dkv_kernel(
    const bf16raw* __restrict__ Q, const bf16raw* __restrict__ K, const bf16raw* __restrict__ V,
    const bf16raw* __restrict__ dO, const float* __restrict__ LSE, const float* __restrict__ Dl,
    int S, int H, int Hkv, int64_t T, float* __restrict__ dK, float* __restrict__ dV,
    int p_bits, const float4* __restrict__ pstat, const float2* __restrict__ dmm) {
  constexpr int KS = DH / 32, JD = DH / 16, NR = AT * DH / 8 / ANT;
  __shared__ uint4 sQ[AT * DH / 8];
  __shared__ uint4 sdO[AT * DH / 8];
  __shared__ __attribute__((aligned(16))) bf16raw sP[4][AT * TS];
  __shared__ __attribute__((aligned(16))) bf16raw sH[4][AT * TS];
  __shared__ __attribute__((aligned(16))) bf16raw sLo[4][AT * TS];
  __shared__ float sL[AT], sD[AT];
  // QP: per query row h, 1/h, z of Q_a, the routed max / min gradients and
  // the indices that take them
  __shared__ float sQh[QP ? AT : 1], sQr[QP ? AT : 1], sQz[QP ? AT : 1];
  __shared__ float sDmx[QP ? AT : 1], sDmn[QP ? AT : 1];
  __shared__ int sAmx[QP ? AT : 1], sAmn[QP ? AT : 1];
  const float qmax = QP ? float((1 << p_bits) - 1) : 0.0f;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int fr = lane & 15, fk = lane >> 4;
  const int ntile = S / AT;
  const int kt = int(blockIdx.x), g = blockIdx.y, b = blockIdx.z;
  const int grp = H / Hkv;
  const int nq = ntile - kt;                           // query tiles at or after this key tile
  const int n_it = grp * nq;
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

  // registers holding the next (query head, query tile)'s Q, dO, LSE and D
  u32x4_t qr[NR], dr[NR];
  float lr = 0.f, dlr = 0.f;
  float4 psr{};
  float2 dmr{};
  auto fetch = [&](int it) {
    const int hq = g * grp + it / nq, qt = kt + it % nq;
    const int64_t qrow0 = row0 + int64_t(qt) * AT;
    tile_to_regs<DH>(qr, Q + qrow0 * ldq + int64_t(hq) * DH, ldq, tid);
    tile_to_regs<DH>(dr, dO + qrow0 * ldq + int64_t(hq) * DH, ldq, tid);
    if (tid < AT) {
      lr = LSE[int64_t(hq) * T + qrow0 + tid];
      dlr = Dl[int64_t(hq) * T + qrow0 + tid];
      if constexpr (QP) {
        psr = pstat[int64_t(hq) * T + qrow0 + tid];
        dmr = dmm[int64_t(hq) * T + qrow0 + tid];
      }
    }
  };
  fetch(0);
  bf16raw* tp = sP[wave];
  bf16raw* th = sH[wave];
  bf16raw* tl = sLo[wave];
  for (int it = 0; it < n_it; ++it) {
    const int qt = kt + it % nq;
    __syncthreads();
    regs_to_k<DH>(sQ, qr, tid);
    regs_to_k<DH>(sdO, dr, tid);
    if (tid < AT) {
      sL[tid] = lr;
      sD[tid] = dlr;
      if constexpr (QP) {
        const QParams prm = make_qparams(psr.x, psr.y, 1.0f, 1.0f, qmax);
        sQh[tid] = prm.h;
        sQr[tid] = prm.r;
        sQz[tid] = prm.z;
        sDmx[tid] = dmr.x;
        sDmn[tid] = dmr.y;
        sAmx[tid] = __float_as_int(psr.z);
        sAmn[tid] = __float_as_int(psr.w);
      }
    }
    __syncthreads();
    fetch(it + 1 < n_it ? it + 1 : it);                 // in flight meanwhile
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
    const bool diag = qt == kt;
#pragma unroll
    for (int jn = 0; jn < 4; ++jn) {
      const int ql = 16 * jn + fr;
      const float L = sL[ql], D = sD[ql];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float p = __builtin_amdgcn_exp2f(fmaf(st[jn][r], sc, -L));
        if (diag && 16 * wave + 4 * fk + r > ql) p = 0.0f;
        if constexpr (QP) {
          QParams prm{};
          prm.h = sQh[ql];
          prm.r = sQr[ql];
          prm.z = sQz[ql];
          const QElem qe = quant_elem(p, prm, qmax);
          const int key = key_w + 4 * fk + r;
          float g = qe.m ? dp[jn][r] : 0.0f;
          if (key == sAmx[ql]) g += sDmx[ql];
          if (key == sAmn[ql]) g += sDmn[ql];
          st[jn][r] = dequant(qe.q, prm);               // P^ enters dV
          dp[jn][r] = p * (g - D) * rs;
        } else {
          st[jn][r] = p;
          dp[jn][r] = p * (dp[jn][r] - D) * rs;         // dS^T (with the 1/sqrt(d) of the logits)
        }
      }
      // P^T query-major: row = query, four consecutive keys
      t16_put4(tp, ql, 4 * fk, st[jn][0], st[jn][1], st[jn][2], st[jn][3]);
      // dS^T as two bf16 terms (hi + lo, 16 significant bits): a component
      // shared by all queries' Q rows would otherwise meet the rounding of dS
      float hi[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) hi[r] = bf2f(f2bf(dp[jn][r]));
      t16_put4(th, ql, 4 * fk, hi[0], hi[1], hi[2], hi[3]);
      t16_put4(tl, ql, 4 * fk, dp[jn][0] - hi[0], dp[jn][1] - hi[1], dp[jn][2] - hi[2],
               dp[jn][3] - hi[3]);
    }
    // dV += P^T dO and dK += dS^T Q: A = rows of keys, k = queries; B = dO^T
    // and Q^T (rows of d), read transposed from the row-major tiles
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      const bf16x8_t ap = t16_frag(tp, 32 * k2, lane);
      const bf16x8_t ah = t16_frag(th, 32 * k2, lane);
      const bf16x8_t al = t16_frag(tl, 32 * k2, lane);
#pragma unroll
      for (int j = 0; j < JD; ++j) {
        adv[j] = mfma(ap, col_frag<DH>(sdO, 32 * k2, 16 * j, lane), adv[j]);
        const bf16x8_t bq = col_frag<DH>(sQ, 32 * k2, 16 * j, lane);
        adk[j] = mfma(al, bq, mfma(ah, bq, adk[j]));
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

// dQ: one workgroup per 64-query tile and head, four waves of 16 queries.  A
// first sweep over the key tiles forms D = sum_j P_ij dP_ij from the very
// probabilities the gradients use (so every row of dS sums to zero to fp32
// rounding) and writes it for the dK/dV kernel; the second sweep accumulates
// dQ = dS K, dS staged key-major as two bf16 terms.
// QP (softmax quantisation): the first sweep also forms Q_a's row sums
// S_h = sum dP^ ((q - z) - m u), S_z = sum dP^ (1 - m) and E = sum P m dP^,
// hence the row's max / min gradients (written to dmm for the dK/dV kernel)
// and D = E + max dmax + min dmin; the second sweep's dP follows Q_a's
// straight-through rule.
template <int DH, bool QP>
__global__ __launch_bounds__(ANT, 2) void attn_bwd_dq_kernel(
    const bf16raw* __restrict__ Q, const bf16raw* __restrict__ K, const bf16raw* __restrict__ V,
    const bf16raw* __restrict__ dO, const float* __restrict__ LSE, float* __restrict__ Dl,
    int S, int H, int Hkv, int64_t T, float* __restrict__ dQ, int p_bits,
    const float4* __restrict__ pstat, float2* __restrict__ dmm) {
  constexpr int KS = DH / 32, JD = DH / 16, NR = AT * DH / 8 / ANT;
  __shared__ uint4 sK[AT * DH / 8];
  __shared__ uint4 sV[AT * DH / 8];
  __shared__ __attribute__((aligned(16))) bf16raw sH[4][AT * TS];
  __shared__ __attribute__((aligned(16))) bf16raw sLo[4][AT * TS];
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
  // QP: per row of this wave, (1/h, z, index of the max, index of the min)
  // and the max / min gradients once sweep 1 has them, in LDS (not registers)
  __shared__ float4 sRq[QP ? 4 : 1][16];
  __shared__ float2 sRg[QP ? 4 : 1][16];
  const float qmax = QP ? float((1 << p_bits) - 1) : 0.0f;
  float sh[QP ? 4 : 1], sz[QP ? 4 : 1];
  if constexpr (QP) {
#pragma unroll
    for (int r = 0; r < 4; ++r) sh[r] = sz[r] = 0.f;
    if (lane < 16) {
      const float4 p4 = pstat[int64_t(h) * T + row0 + q_w + lane];
      const QParams pr = make_qparams(p4.x, p4.y, 1.0f, 1.0f, qmax);
      sRq[wave][lane] = make_float4(pr.r, pr.z, p4.z, p4.w);
    }
  }
  f32x4_t adq[JD];
#pragma unroll
  for (int j = 0; j < JD; ++j) adq[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  u32x4_t kr[NR], vr[NR];
  const int nk = qt + 1;
  auto fetch = [&](int t) {
    const int64_t krow = row0 + int64_t(t) * AT;
    tile_to_regs<DH>(kr, K + krow * ldk + int64_t(g) * DH, ldk, tid);
    tile_to_regs<DH>(vr, V + krow * ldk + int64_t(g) * DH, ldk, tid);
  };
  fetch(0);
  bf16raw* th = sH[wave];
  bf16raw* tl = sLo[wave];
  for (int it = 0; it < 2 * nk; ++it) {
    const int kt = it < nk ? it : it - nk;
    __syncthreads();
    regs_to_k<DH>(sK, kr, tid);
    regs_to_k<DH>(sV, vr, tid);
    __syncthreads();
    fetch(kt + 1 < nk ? kt + 1 : 0);                    // in flight meanwhile
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
    const bool diag = kt == qt;
#pragma unroll
    for (int jn = 0; jn < 4; ++jn)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float p = __builtin_amdgcn_exp2f(fmaf(st[jn][r], sc, -lse[r]));
        if (diag && 16 * jn + fr > 16 * wave + 4 * fk + r) p = 0.0f;
        st[jn][r] = p;
      }
    if (it < nk) {
      // sweep 1: D (with QP, Q_a's row sums first)
#pragma unroll
      for (int jn = 0; jn < 4; ++jn)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          if constexpr (QP) {
            const float4 rq = sRq[wave][4 * fk + r];
            QParams pr{};
            pr.r = rq.x;
            pr.z = rq.y;
            const QElem qe = quant_elem(st[jn][r], pr, qmax);
            const float t = qe.q - pr.z;
            sh[r] += dp[jn][r] * (qe.m ? t - qe.u : t);
            sz[r] += qe.m ? 0.0f : dp[jn][r];
            dl[r] += qe.m ? st[jn][r] * dp[jn][r] : 0.0f;
          } else {
            dl[r] += st[jn][r] * dp[jn][r];
          }
        }
      if (it == nk - 1) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
#pragma unroll
          for (int o = 1; o < 16; o <<= 1) dl[r] += __shfl_xor(dl[r], o);
          if constexpr (QP) {
#pragma unroll
            for (int o = 1; o < 16; o <<= 1) {
              sh[r] += __shfl_xor(sh[r], o);
              sz[r] += __shfl_xor(sz[r], o);
            }
            const int64_t ri = int64_t(h) * T + row0 + q_w + 4 * fk + r;
            const float4 p4 = pstat[ri];
            const QParams pr = make_qparams(p4.x, p4.y, 1.0f, 1.0f, qmax);
            const QGrad qg = quant_group_grad(sh[r], sz[r], p4.x, p4.y, pr, qmax);
            dl[r] += p4.x * qg.dmx + p4.y * qg.dmn;
            if (fr == 0) {
              sRg[wave][4 * fk + r] = make_float2(qg.dmx, qg.dmn);
              dmm[ri] = make_float2(qg.dmx, qg.dmn);
            }
          }
        }
        if (fr == 0) {
#pragma unroll
          for (int r = 0; r < 4; ++r) Dl[int64_t(h) * T + row0 + q_w + 4 * fk + r] = dl[r];
        }
      }
      continue;
    }
    // sweep 2: dS = P (dP - D) / sqrt(d), key-major as hi + lo bf16 terms: each
    // row of dS sums to zero, so a component shared by all K rows cancels in
    // the exact product and must not survive the rounding of dS
#pragma unroll
    for (int jn = 0; jn < 4; ++jn) {
      float v[4], hi[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float gp = dp[jn][r];
        if constexpr (QP) {
          const float4 rq = sRq[wave][4 * fk + r];
          const float2 rg = sRg[wave][4 * fk + r];
          QParams pr{};
          pr.r = rq.x;
          pr.z = rq.y;
          const QElem qe = quant_elem(st[jn][r], pr, qmax);
          const int key = kt * AT + 16 * jn + fr;
          gp = qe.m ? gp : 0.0f;
          if (key == __float_as_int(rq.z)) gp += rg.x;
          if (key == __float_as_int(rq.w)) gp += rg.y;
        }
        v[r] = st[jn][r] * (gp - dl[r]) * rs;
        hi[r] = bf2f(f2bf(v[r]));
      }
      t16_put4(th, 16 * jn + fr, 4 * fk, hi[0], hi[1], hi[2], hi[3]);
      t16_put4(tl, 16 * jn + fr, 4 * fk, v[0] - hi[0], v[1] - hi[1], v[2] - hi[2], v[3] - hi[3]);
    }
    // dQ += dS K: A = dS rows (queries), k = keys; B = K^T rows (d)
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      const bf16x8_t ah = t16_frag(th, 32 * k2, lane);
      const bf16x8_t al = t16_frag(tl, 32 * k2, lane);
#pragma unroll
      for (int j = 0; j < JD; ++j) {
        const bf16x8_t bk = col_frag<DH>(sK, 32 * k2, 16 * j, lane);
        adq[j] = mfma(al, bk, mfma(ah, bk, adq[j]));
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
                      int Hkv, int p_bits, float* O, float* LSE, float4* pstat, hipStream_t st) {
  const dim3 grid(unsigned(S / AT), unsigned(H), unsigned(T / S));
  const auto q = static_cast<const bf16raw*>(Q);
  const auto k = static_cast<const bf16raw*>(K);
  const auto v = static_cast<const bf16raw*>(V);
  if (p_bits < 16)
    hipLaunchKernelGGL(attn_fwd_q_kernel<DH>, grid, dim3(ANT), 0, st, q, k, v, S, H, Hkv, p_bits,
                       O, LSE, pstat, T);
  else if (S % (2 * AT) == 0)
    hipLaunchKernelGGL(attn_fwd2_kernel<DH>, dim3(unsigned(S / (2 * AT)), unsigned(H), unsigned(T / S)),
                       dim3(ANT), 0, st, q, k, v, S, H, Hkv, O, LSE, T);
  else
    hipLaunchKernelGGL(attn_fwd_kernel<DH>, grid, dim3(ANT), 0, st, q, k, v, S, H, Hkv, O, LSE, T);
  return hipGetLastError();
}

template <int DH, bool QP>
void attn_bwd_launch(const void* Q, const void* K, const void* V, const void* dO,
                     const float* LSE, const float4* pstat, int64_t T, int S, int H, int Hkv,
                     int p_bits, float* Dl, float2* dmm, float* dQ, float* dK, float* dV,
                     hipStream_t st) {
  const auto q = static_cast<const bf16raw*>(Q);
  const auto k = static_cast<const bf16raw*>(K);
  const auto v = static_cast<const bf16raw*>(V);
  const auto o = static_cast<const bf16raw*>(dO);
  // dQ first: it also writes D (and, quantised, the max / min gradients),
  // which the dK/dV kernel reads
  hipLaunchKernelGGL((attn_bwd_dq_kernel<DH, QP>), dim3(unsigned(S / AT), unsigned(H), unsigned(T / S)),
                     dim3(ANT), 0, st, q, k, v, o, LSE, Dl, S, H, Hkv, T, dQ, p_bits, pstat, dmm);
  hipLaunchKernelGGL((attn_bwd_dkv_kernel<DH, QP>), dim3(unsigned(S / AT), unsigned(Hkv), unsigned(T / S)),
                     dim3(ANT), 0, st, q, k, v, o, LSE, Dl, S, H, Hkv, T, dK, dV, p_bits, pstat,
                     dmm);
}

template <int DH>
hipError_t attn_bwd_t(const void* Q, const void* K, const void* V, const void* dO,
                      const float* LSE, const float4* pstat, int64_t T, int S, int H, int Hkv,
                      int p_bits, float* ws, float* dQ, float* dK, float* dV, hipStream_t st) {
  float2* dmm = reinterpret_cast<float2*>(ws + T * H);
  if (p_bits < 16)
    attn_bwd_launch<DH, true>(Q, K, V, dO, LSE, pstat, T, S, H, Hkv, p_bits, ws, dmm, dQ, dK, dV, st);
  else
    attn_bwd_launch<DH, false>(Q, K, V, dO, LSE, nullptr, T, S, H, Hkv, 16, ws, nullptr, dQ, dK, dV,
                               st);
  return hipGetLastError();
}

}  // namespace

bool attn_supported(int64_t T, int S, int H, int Hkv, int dh) {
  return (dh == 64 || dh == 128) && S > 0 && S % AT == 0 && T > 0 && T % S == 0 && H > 0 &&
         Hkv > 0 && H % Hkv == 0 && T / S <= 65535 && H <= 65535;
}

size_t attn_bwd_ws_floats(int64_t T, int H, int p_bits) {
  return size_t(T) * size_t(H) * (p_bits < 16 ? 3 : 1);
}

hipError_t attn_fwd(const void* Q, const void* K, const void* V, int64_t T, int S, int H, int Hkv,
                    int dh, int p_bits, float* O, float* LSE, float* pstat, hipStream_t st) {
  if (!attn_supported(T, S, H, Hkv, dh)) return hipErrorInvalidValue;
  float4* ps = reinterpret_cast<float4*>(pstat);
  return dh == 128 ? attn_fwd_t<128>(Q, K, V, T, S, H, Hkv, p_bits, O, LSE, ps, st)
                   : attn_fwd_t<64>(Q, K, V, T, S, H, Hkv, p_bits, O, LSE, ps, st);
}

hipError_t attn_bwd(const void* Q, const void* K, const void* V, const void* dO, const float* LSE,
                    const float* pstat, int64_t T, int S, int H, int Hkv, int dh, int p_bits,
                    float* ws, float* dQ, float* dK, float* dV, hipStream_t st) {
  if (!attn_supported(T, S, H, Hkv, dh)) return hipErrorInvalidValue;
  const float4* ps = reinterpret_cast<const float4*>(pstat);
  return dh == 128 ? attn_bwd_t<128>(Q, K, V, dO, LSE, ps, T, S, H, Hkv, p_bits, ws, dQ, dK, dV, st)
                   : attn_bwd_t<64>(Q, K, V, dO, LSE, ps, T, S, H, Hkv, p_bits, ws, dQ, dK, dV, st);
}

}  // namespace oq
