// Quantiser kernels: learnable weight clipping (Eq. 2) and per-token MinMax
// activation fake-quant with the LET input transform (Eq. 3-4), forward and
// straight-through backward.
//
// Work layout: a workgroup of 256 threads walks R consecutive rows.  A row is
// split into 8-element chunks (16-byte bf16 / 32-byte fp32 vectors); thread t
// owns chunks t, t+256, t+512, ... of every row, so per-column running sums
// (the LET scale gradient) stay in registers across the R rows and every
// global access is a coalesced 16/32-byte vector.
//  * small groups (g a power of two <= 512): a group is g/8 consecutive lanes
//    of one wave; its max/min (with the lowest index) and its gradient sums
//    are xor-butterflies over those lanes;
//  * whole-row groups (per output channel / per token): wave butterflies,
//    then the four wave results combined in a fixed order through LDS.
// Every reduction has a fixed shape, so results are bitwise reproducible.
#include <float.h>
#include <algorithm>
#include <type_traits>
#include <limits.h>
#include <mutex>
#include <vector>

#include "common.h"
#include "oq_internal.h"

namespace oq {
namespace {

constexpr int NT = 256;

struct MinMax {
  float mx, mn;
  int imx, imn;
};

OQ_DEV MinMax minmax_init() { return MinMax{-FLT_MAX, FLT_MAX, INT_MAX, INT_MAX}; }
OQ_DEV void minmax_add(MinMax& s, float v, int idx) {
  sel_max(s.mx, s.imx, v, idx);
  sel_min(s.mn, s.imn, v, idx);
}

// Whole-workgroup (max, argmax, min, argmin); every thread gets the result.
template <int NTB = NT>
OQ_DEV MinMax block_minmax(MinMax v, MinMax* sh) {
  group_minmax<64>(v.mx, v.imx, v.mn, v.imn);
  const int wave = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[wave] = v;
  __syncthreads();
  MinMax r = sh[0];
#pragma unroll
  for (int w = 1; w < NTB / 64; ++w) {
    sel_max(r.mx, r.imx, sh[w].mx, sh[w].imx);
    sel_min(r.mn, r.imn, sh[w].mn, sh[w].imn);
  }
  return r;
}

OQ_DEV float2 block_sum2(float2 v, float2* sh) {
  v.x = group_sum<64>(v.x);
  v.y = group_sum<64>(v.y);
  const int wave = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[wave] = v;
  __syncthreads();
  float2 r = sh[0];
#pragma unroll
  for (int w = 1; w < NT / 64; ++w) {
    r.x += sh[w].x;
    r.y += sh[w].y;
  }
  return r;
}

// Workgroup barrier that waits for LDS traffic only: global loads issued
// before it (the next row's prefetch) stay in flight across it.
OQ_DEV void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Register image of 8 consecutive elements as loaded (bf16 packed or fp32).
template <typename TX>
struct Chunk8 {
  static constexpr int NV = sizeof(TX) == 2 ? 1 : 2;
  uint4 v[NV];
  OQ_DEV void load(const TX* p) {
#pragma unroll
    for (int i = 0; i < NV; ++i) v[i] = reinterpret_cast<const uint4*>(p)[i];
  }
  OQ_DEV static uint32_t word(const uint4& q, int k) {
    return k == 0 ? q.x : (k == 1 ? q.y : (k == 2 ? q.z : q.w));
  }
  OQ_DEV float at(int e) const {
    const uint4& q = v[sizeof(TX) == 2 ? 0 : e >> 2];
    if constexpr (sizeof(TX) == 2) {
      const uint32_t w = word(q, e >> 1);
      return __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
    } else {
      return __uint_as_float(word(q, e & 3));
    }
  }
};

// ------------------------------------------------------------------ LWC forward
template <typename TW, typename TQ, int KC, bool WHOLE_ROW>
__global__ __launch_bounds__(NT) void lwc_fwd_kernel(
    const TW* __restrict__ W, int64_t c_out, int64_t c_in, const float* __restrict__ s,
    const float* __restrict__ gl, const float* __restrict__ bl, int bits, int group, int R,
    TQ* __restrict__ wdq, uint8_t* __restrict__ codes, float* __restrict__ hout,
    float* __restrict__ zout, int quant) {
  __shared__ MinMax shm[NT / 64];
  const int tid = threadIdx.x;
  const int cpr = int(c_in / 8);
  const int ng = int(c_in / group);
  const int L = group / 8;
  const float qmax = float((1 << bits) - 1);

  float sv[KC][8];
#pragma unroll
  for (int k = 0; k < KC; ++k) {
    const int j = tid + NT * k;
#pragma unroll
    for (int e = 0; e < 8; ++e) sv[k][e] = 1.0f;
    if (s && j < cpr) load8(s + 8 * j, sv[k]);
  }

  const int64_t r0 = int64_t(blockIdx.x) * R;
  const int64_t r1 = min(c_out, r0 + R);
  for (int64_t row = r0; row < r1; ++row) {
    const TW* wrow = W + row * c_in;
    if constexpr (WHOLE_ROW) {
      float v[KC][8];
      MinMax st = minmax_init();
#pragma unroll
      for (int k = 0; k < KC; ++k) {
        const int j = tid + NT * k;
        if (j < cpr) {
          load8(wrow + 8 * j, v[k]);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            if (s) v[k][e] = v[k][e] * sv[k][e];
            minmax_add(st, v[k][e], 8 * j + e);
          }
        }
      }
      st = block_minmax(st, shm);
      const QParams p = make_group_qparams(quant, st.mx, st.mn, gl[row], bl[row], qmax);
#pragma unroll
      for (int k = 0; k < KC; ++k) {
        const int j = tid + NT * k;
        if (j < cpr) {
          float q[8], d[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            q[e] = quant_elem(v[k][e], p, qmax).q;
            d[e] = dequant(q[e], p);
          }
          if (wdq) store8(wdq + row * c_in + 8 * j, d);
          if (codes) store8_codes(codes + row * c_in + 8 * j, q);
        }
      }
      if (tid == 0) {
        if (hout) hout[row] = p.h;
        if (zout) zout[row] = p.z;
      }
    } else {
#pragma unroll
      for (int k = 0; k < KC; ++k) {
        const int j = tid + NT * k;
        const bool valid = j < cpr;
        float v[8];
        MinMax st = minmax_init();
        if (valid) {
          load8(wrow + 8 * j, v);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            if (s) v[e] = v[e] * sv[k][e];
            minmax_add(st, v[e], 8 * j + e);
          }
        }
        dyn_group_minmax(st.mx, st.imx, st.mn, st.imn, L);
        if (valid) {
          const int grp = j / L;
          const QParams p = make_group_qparams(quant, st.mx, st.mn, gl[row * ng + grp],
                                               bl[row * ng + grp], qmax);
          float q[8], d[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            q[e] = quant_elem(v[e], p, qmax).q;
            d[e] = dequant(q[e], p);
          }
          if (wdq) store8(wdq + row * c_in + 8 * j, d);
          if (codes) store8_codes(codes + row * c_in + 8 * j, q);
          if (j % L == 0) {
            if (hout) hout[row * ng + grp] = p.h;
            if (zout) zout[row * ng + grp] = p.z;
          }
        }
      }
    }
  }
}

// ------------------------------------------------------------------ LWC backward
// Per group:  S_h = sum g*((q - z) - m*u),  S_z = sum g*(1 - m)  ->  dgamma, dbeta
// per element: dW~ = g*m + [i = argmax] dmax + [i = argmin] dmin
// per column (optional): partial sum over this block's rows of dW~ * W.
template <typename TW, int KC, bool WHOLE_ROW, bool LETW, int NTB = NT>
__global__ __launch_bounds__(NTB) void lwc_bwd_kernel(
    const TW* __restrict__ W, int64_t c_out, int64_t c_in, const float* __restrict__ s,
    const float* __restrict__ gl, const float* __restrict__ bl, int bits, int group, int R,
    const float* __restrict__ dW, float* __restrict__ dgl, float* __restrict__ dbl,
    float* __restrict__ dWt, float* __restrict__ ds_parts, int quant, float gs) {
  __shared__ MinMax shm[NTB / 64];
  __shared__ float2 shs[NTB / 64];
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int cpr = int(c_in / 8);
  const int ng = int(c_in / group);
  const int L = group / 8;
  const float qmax = float((1 << bits) - 1);

  // LETW: s is given or its partials are wanted (the weight-path LET scale,
  // ones when s is absent, and the ds partials)
  constexpr int KS = LETW ? KC : 1;
  float sv[KS][8], dsacc[KS][8];
#pragma unroll
  for (int k = 0; k < KS; ++k) {
    const int j = tid + NTB * k;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      sv[k][e] = 1.0f;
      dsacc[k][e] = 0.0f;
    }
    if (LETW && s && j < cpr) load8(s + 8 * j, sv[k]);
  }

  const int64_t r0 = int64_t(blockIdx.x) * R;
  const int64_t r1 = min(c_out, r0 + R);
  // whole rows of up to two chunks per thread: the next row's W and dW^ are
  // loaded while this row is reduced (wider rows would spill)
  constexpr bool PF = WHOLE_ROW && KC <= (NTB >= 512 ? 4 : 2);
  Chunk8<TW> wn[KC];
  float gn[KC][8];
  auto issue = [&](int64_t row) {
#pragma unroll
    for (int k = 0; k < KC; ++k) {
      const int j = tid + NTB * k;
      if (j < cpr) {
        wn[k].load(W + row * c_in + 8 * j);
        load8(dW + row * c_in + 8 * j, gn[k]);
      }
    }
  };
  if constexpr (PF) {
    if (r0 < r1) issue(r0);
  }
  for (int64_t row = r0; row < r1; ++row) {
    const TW* wrow = W + row * c_in;
    const float* grow = dW + row * c_in;
    if constexpr (WHOLE_ROW) {
      // the row stays packed as loaded; w~ is recomputed in each pass
      Chunk8<TW> wc[KC];
      float g[KC][8];
      MinMax st = minmax_init();
      if constexpr (PF) {
#pragma unroll
        for (int k = 0; k < KC; ++k) {
          wc[k] = wn[k];
#pragma unroll
          for (int e = 0; e < 8; ++e) g[k][e] = gn[k][e];
        }
        if (row + 1 < r1) issue(row + 1);
      } else {
#pragma unroll
        for (int k = 0; k < KC; ++k) {
          const int j = tid + NTB * k;
          if (j < cpr) {
            wc[k].load(wrow + 8 * j);
            load8(grow + 8 * j, g[k]);
          }
        }
      }
      auto wt_at = [&](int k, int e) {
        const float w = wc[k].at(e);
        if constexpr (LETW) return w * sv[k][e];
        else return w;
      };
#pragma unroll
      for (int k = 0; k < KC; ++k) {
        const int j = tid + NTB * k;
        if (j < cpr) {
#pragma unroll
          for (int e = 0; e < 8; ++e) minmax_add(st, wt_at(k, e), 8 * j + e);
        }
      }
      wave_minmax(st.mx, st.imx, st.mn, st.imn);
      if ((tid & 63) == 0) shm[wave] = st;
      lds_barrier();
      st = shm[0];
#pragma unroll
      for (int w8 = 1; w8 < NTB / 64; ++w8) {
        sel_max(st.mx, st.imx, shm[w8].mx, shm[w8].imx);
        sel_min(st.mn, st.imn, shm[w8].mn, shm[w8].imn);
      }
      const QParams p = make_group_qparams(quant, st.mx, st.mn, gl[row], bl[row], qmax);
      float2 sums = make_float2(0.f, 0.f);
#pragma unroll
      for (int k = 0; k < KC; ++k) {
        const int j = tid + NTB * k;
        if (j < cpr) {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            group_terms(quant, g[k][e], quant_elem(wt_at(k, e), p, qmax), p, qmax, sums.x, sums.y);
        }
      }
      sums.x = wave_sum(sums.x);
      sums.y = wave_sum(sums.y);
      if ((tid & 63) == 0) shs[wave] = sums;
      lds_barrier();
      sums = shs[0];
#pragma unroll
      for (int w8 = 1; w8 < NTB / 64; ++w8) {
        sums.x += shs[w8].x;
        sums.y += shs[w8].y;
      }
      const GroupGrad qg = group_param_grads(quant, sums.x, sums.y, st.mx, st.mn, p, qmax, gs);
      if (tid == 0) {
        dgl[row] = qg.d1;
        dbl[row] = qg.d2;
      }
      if (LETW || dWt) {
#pragma unroll
        for (int k = 0; k < KC; ++k) {
          const int j = tid + NTB * k;
          if (j < cpr) {
            // without LET only dW~ needs this pass: dW^ is read again rather
            // than kept live through the reductions
            float gg[8], d[8];
            if constexpr (LETW) {
#pragma unroll
              for (int e = 0; e < 8; ++e) gg[e] = g[k][e];
            } else {
              load8(grow + 8 * j, gg);
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const int col = 8 * j + e;
              float x = quant_elem(wt_at(k, e), p, qmax).m ? gg[e] : 0.0f;
              if (quant == WQ_LWC) {
                if (col == st.imx) x += qg.dmx;
                if (col == st.imn) x += qg.dmn;
              }
              d[e] = x;
              if constexpr (LETW) dsacc[k][e] += x * wc[k].at(e);
            }
            if (dWt) store8(dWt + row * c_in + 8 * j, d);
          }
        }
      }
    } else {
#pragma unroll
      for (int k = 0; k < KC; ++k) {
        const int j = tid + NTB * k;
        const bool valid = j < cpr;
        float w[8], wt[8], g[8];
        MinMax st = minmax_init();
        if (valid) {
          load8(wrow + 8 * j, w);
          load8(grow + 8 * j, g);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            if constexpr (LETW) wt[e] = w[e] * sv[k][e];
            else wt[e] = w[e];
            minmax_add(st, wt[e], 8 * j + e);
          }
        }
        dyn_group_minmax(st.mx, st.imx, st.mn, st.imn, L);
        const int grp = j / L;
        QParams p{};
        float sh = 0.f, sz = 0.f;
        bool mk[8];
        if (valid) {
          p = make_group_qparams(quant, st.mx, st.mn, gl[row * ng + grp], bl[row * ng + grp], qmax);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const QElem qe = quant_elem(wt[e], p, qmax);
            mk[e] = qe.m;
            group_terms(quant, g[e], qe, p, qmax, sh, sz);
          }
        }
        sh = dyn_group_sum(sh, L);
        sz = dyn_group_sum(sz, L);
        if (valid) {
          const GroupGrad qg = group_param_grads(quant, sh, sz, st.mx, st.mn, p, qmax, gs);
          if (j % L == 0) {
            dgl[row * ng + grp] = qg.d1;
            dbl[row * ng + grp] = qg.d2;
          }
          float d[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int col = 8 * j + e;
            float x = mk[e] ? g[e] : 0.0f;
            if (quant == WQ_LWC) {
              if (col == st.imx) x += qg.dmx;
              if (col == st.imn) x += qg.dmn;
            }
            d[e] = x;
            if constexpr (LETW) dsacc[k][e] += x * w[e];
          }
          if (dWt) store8(dWt + row * c_in + 8 * j, d);
        }
      }
    }
  }
  if (LETW && ds_parts) {
#pragma unroll
    for (int k = 0; k < KS; ++k) {
      const int j = tid + NTB * k;
      if (j < cpr) store8(ds_parts + int64_t(blockIdx.x) * c_in + 8 * j, dsacc[k]);
    }
  }
}

// ------------------------------------------------------------------ LWC backward, lane-owned runs
// Groups of at most 512 weights without LET scaling: each lane owns a run of
// E consecutive weights of one row (E / 8 independent 16-byte loads in
// flight, with the run's gradient), takes the run's max / min (and the first
// index holding each where dW~ is wanted), and combines with the other
// group / E lanes of its group (adjacent, aligned lanes) by butterflies.  The
// group parameters are then computed once per E weights instead of once per
// 8, and the kernel has no divergent branches.  A tail lane past the last run
// repeats the last run without storing, so every butterfly sees whole groups.
// (The same layout for the forward, with E = 128, left each 16-byte access of
// a wave 256 bytes from the next; the forward below walks coalesced chunks.)

// Register image of a run of E elements as 16-byte vectors.
template <typename TW, int E>
struct Run {
  static constexpr int NV = sizeof(TW) == 2 ? E / 8 : E / 4;
  uint4 v[NV];
  OQ_DEV void load(const TW* p) {
#pragma unroll
    for (int i = 0; i < NV; ++i) v[i] = reinterpret_cast<const uint4*>(p)[i];
  }
  OQ_DEV static uint32_t word(const uint4& q, int k) {
    return k == 0 ? q.x : (k == 1 ? q.y : (k == 2 ? q.z : q.w));
  }
  OQ_DEV float at(int i) const {
    if constexpr (sizeof(TW) == 2) {
      const uint32_t w = word(v[i >> 3], (i >> 1) & 3);
      return __uint_as_float((i & 1) ? (w & 0xffff0000u) : (w << 16));
    } else {
      return __uint_as_float(word(v[i >> 2], i & 3));
    }
  }
};

// max / min of a run (values only: the forward parameters need no index)
template <typename TW, int E>
OQ_DEV void run_range(const Run<TW, E>& x, float& mx, float& mn) {
  mx = x.at(0);
  mn = mx;
#pragma unroll
  for (int i = 1; i < E; ++i) {
    mx = fmaxf(mx, x.at(i));
    mn = fminf(mn, x.at(i));
  }
}

// Index (within the row) of the first element of the run equal to v.
template <typename TW, int E>
OQ_DEV int run_first(const Run<TW, E>& x, int col0, float v) {
  int idx = E - 1;
#pragma unroll
  for (int i = E - 2; i >= 0; --i) idx = x.at(i) == v ? i : idx;
  return col0 + idx;
}

// (max, min) over the L aligned lanes of a group, values only.
OQ_DEV void dyn_group_range(float& mx, float& mn, int L) {
  for (int off = 1; off < L; off <<= 1) {
    mx = fmaxf(mx, __shfl_xor(mx, off));
    mn = fminf(mn, __shfl_xor(mn, off));
  }
}

// ------------------------------------------------------------------ LWC forward, coalesced
// Power-of-two groups of at most 512 weights without LET scaling.  The matrix
// is walked as a flat sequence of 8-weight chunks (groups never straddle a
// row); lane l of a wave takes chunk 64 u + l of each of its U slices, so
// every load and store of a wave is 1 KiB of contiguous memory.  A group is
// G = group / 8 adjacent lanes: their max / min combine by butterflies.  The
// group parameters (sigmoids in fp64, Eq. 2's h, 1/h, z) are computed once
// per group by an owner lane: the U * 64 / G groups of a wave step are owned
// by lanes 0, 1, ... in order, which fetch their group's range and hand back
// h, 1/h, z through cross-lane reads.  Lanes past the last chunk repeat it
// without storing (whole groups, since a row holds whole groups).
template <typename TW>
OQ_DEV void load_chunk(const TW* p, float (&x)[8]) {
  if constexpr (sizeof(TW) == 2) {
    const uint4 q = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int e = 0; e < 8; ++e)
      x[e] = __uint_as_float((e & 1) ? (w[e >> 1] & 0xffff0000u) : (w[e >> 1] << 16));
  } else {
    const float4 a = reinterpret_cast<const float4*>(p)[0];
    const float4 b = reinterpret_cast<const float4*>(p)[1];
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
    x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
  }
}

template <typename TW, typename TQ, int G, bool CODES>
__global__ __launch_bounds__(NT) void lwc_fwd_coal_kernel(
    const TW* __restrict__ W, int64_t nchunk, const float* __restrict__ gl,
    const float* __restrict__ bl, int bits, TQ* __restrict__ wdq, uint8_t* __restrict__ codes,
    float* __restrict__ hout, float* __restrict__ zout, float4* __restrict__ gstat) {
  constexpr int U = G < 8 ? G : 8;           // slices per lane: the owners fit in a wave
  constexpr int NGW = 64 / G;                // groups per slice
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t(blockIdx.x) * NT + threadIdx.x) >> 6;
  const int64_t nwave = (int64_t(gridDim.x) * NT) >> 6;
  const int64_t nstep = (nchunk + 64 * U - 1) / (64 * U);
  const int64_t ngroup = nchunk / G;
  const float qmax = float((1 << bits) - 1);
  for (int64_t step = wave; step < nstep; step += nwave) {
    const int64_t c0 = step * (64 * U) + lane;
    float x[U][8], mx[U], mn[U];
#pragma unroll
    for (int u = 0; u < U; ++u) load_chunk(W + 8 * min(c0 + 64 * u, nchunk - 1), x[u]);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      mx[u] = x[u][0];
      mn[u] = x[u][0];
#pragma unroll
      for (int e = 1; e < 8; ++e) {
        mx[u] = fmaxf(mx[u], x[u][e]);
        mn[u] = fminf(mn[u], x[u][e]);
      }
#pragma unroll
      for (int off = 1; off < G; off <<= 1) {
        mx[u] = fmaxf(mx[u], __shfl_xor(mx[u], off));
        mn[u] = fminf(mn[u], __shfl_xor(mn[u], off));
      }
    }
    // owner lane o holds group step * U * NGW + o: slice o / NGW, lanes
    // (o % NGW) * G .. + G - 1 of it
    float gmx = 0.f, gmn = 0.f;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float a = __shfl(mx[u], (lane % NGW) * G);
      const float b = __shfl(mn[u], (lane % NGW) * G);
      if (lane / NGW == u) {
        gmx = a;
        gmn = b;
      }
    }
    const int64_t g = min(step * (U * NGW) + lane, ngroup - 1);
    float h = 1.f, r = 1.f, z = 0.f;
    if (lane < U * NGW) {
      const QParams p = make_qparams(gmx, gmn, clip_strength(gl[g]), clip_strength(bl[g]), qmax);
      h = p.h;
      r = p.r;
      z = p.z;
      if (step * (U * NGW) + lane < ngroup) {
        if (hout) hout[g] = p.h;
        if (zout) zout[g] = p.z;
        if (gstat) {
          gstat[2 * g] = make_float4(gmx, gmn, p.h, p.z);
          gstat[2 * g + 1] = make_float4(p.gamma, p.beta, p.r, 0.0f);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int own = u * NGW + lane / G;
      const float hu = __shfl(h, own), ru = __shfl(r, own), zu = __shfl(z, own);
      const int64_t c = c0 + 64 * u;
      // rint(u) and z are integers below 2^24, so clamp(rint(u) + z, 0, qmax) - z
      // is exactly med3(rint(u), -z, qmax - z): one instruction for Eq. 2's clamp
      const float lo = -zu, hi = qmax - zu;
      float d[8], q[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float tq = __builtin_amdgcn_fmed3f(rintf(x[u][e] * ru), lo, hi);
        d[e] = tq * hu;
        if constexpr (CODES) q[e] = tq + zu;
      }
      if (c < nchunk) {
        if (wdq) store8(wdq + 8 * c, d);
        if constexpr (CODES) store8_codes(codes + 8 * c, q);
      }
    }
  }
}

template <typename TW, int E, bool DWT>
__global__ __launch_bounds__(NT) void lwc_bwd_run_kernel(
    const TW* __restrict__ W, int64_t c_out, int64_t c_in, const float* __restrict__ gl,
    const float* __restrict__ bl, int bits, int group, const float* __restrict__ dW,
    float* __restrict__ dgl, float* __restrict__ dbl, float* __restrict__ dWt, int parts,
    int64_t part_stride) {
  const uint32_t runs = uint32_t(c_in / E), nrun = uint32_t(c_out) * runs;  // < 2^31 (host)
  uint32_t t = blockIdx.x * NT + threadIdx.x;
  const bool valid = t < nrun;
  if (!valid) t = nrun - 1;
  const uint32_t rq = t / runs;
  const int64_t row = rq;
  const int col0 = int(t - rq * runs) * E;
  const float qmax = float((1 << bits) - 1);

  Run<TW, E> x;
  x.load(W + row * c_in + col0);
  const float* grow = dW + row * c_in + col0;
  Run<float, E> gr;                  // the run's dL/dW^, all loads in flight at once
  gr.load(grow);
  // a K-split product leaves `parts` partial dW^ spaced part_stride apart:
  // summed here in order, ((p0 + p1) + p2) + ...
  for (int q = 1; q < parts; ++q) {
    Run<float, E> pq;
    pq.load(grow + q * part_stride);
#pragma unroll
    for (int i = 0; i < Run<float, E>::NV; ++i) {
      gr.v[i].x = __float_as_uint(__uint_as_float(gr.v[i].x) + __uint_as_float(pq.v[i].x));
      gr.v[i].y = __float_as_uint(__uint_as_float(gr.v[i].y) + __uint_as_float(pq.v[i].y));
      gr.v[i].z = __float_as_uint(__uint_as_float(gr.v[i].z) + __uint_as_float(pq.v[i].z));
      gr.v[i].w = __float_as_uint(__uint_as_float(gr.v[i].w) + __uint_as_float(pq.v[i].w));
    }
  }
  // max / min of the group; with DWT also the lowest index holding each
  // (values first, then the first matching index in the run, then (max,
  // index) across the group's lanes): only dW~ places the max/min gradient
  float mx, mn;
  run_range(x, mx, mn);
  int imx = 0, imn = 0;
  if constexpr (DWT) {
    imx = run_first(x, col0, mx);
    imn = run_first(x, col0, mn);
    if (group > E) dyn_group_minmax(mx, imx, mn, imn, group / E);
  } else {
    if (group > E) dyn_group_range(mx, mn, group / E);
  }
  const int64_t gi = row * (c_in / group) + col0 / group;
  const QParams p = make_qparams(mx, mn, clip_strength(gl[gi]), clip_strength(bl[gi]), qmax);
  // S_h = sum g ((q - z) - m u), S_z = sum g (1 - m): per 8-element chunk, then a tree
  // q - z = med3(rint(u), -z, qmax - z) exactly (integers below 2^24), and the
  // element is inside the clamp (m = 1) exactly when med3 left rint(u) alone
  const float lo = -p.z, hi = qmax - p.z;
  float ph[E / 8], pz[E / 8];
#pragma unroll
  for (int c = 0; c < E / 8; ++c) {
    float sh = 0.f, sz = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float g = gr.at(8 * c + e);
      const float u = x.at(8 * c + e) * p.r;
      const float ru = rintf(u);
      const float tq = __builtin_amdgcn_fmed3f(ru, lo, hi);
      const bool m = tq == ru;
      sh += g * (m ? tq - u : tq);
      sz += m ? 0.0f : g;
    }
    ph[c] = sh;
    pz[c] = sz;
  }
#pragma unroll
  for (int w = 1; w < E / 8; w <<= 1)
#pragma unroll
    for (int c = 0; c < E / 8; c += 2 * w) {
      ph[c] += ph[c + w];
      pz[c] += pz[c + w];
    }
  float sh = ph[0], sz = pz[0];
  if (group > E) {
    sh = dyn_group_sum(sh, group / E);
    sz = dyn_group_sum(sz, group / E);
  }
  const QGrad qg = quant_group_grad(sh, sz, mx, mn, p, qmax);
  if (!valid) return;
  if (col0 % group == 0) {
    dgl[gi] = qg.dgamma * p.gamma * (1.0f - p.gamma);
    dbl[gi] = qg.dbeta * p.beta * (1.0f - p.beta);
  }
  if constexpr (DWT) {
#pragma unroll
    for (int c = 0; c < E / 8; ++c) {
      float d[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int col = col0 + 8 * c + e;
        const float ru = rintf(x.at(8 * c + e) * p.r);
        float v = __builtin_amdgcn_fmed3f(ru, lo, hi) == ru ? gr.at(8 * c + e) : 0.0f;
        if (col == imx) v += qg.dmx;
        if (col == imn) v += qg.dmn;
        d[e] = v;
      }
      store8(dWt + row * c_in + col0 + 8 * c, d);
    }
  }
}

// ------------------------------------------------------------------ activation forward, wave per row
// Token rows of up to 512 * CH elements: each wave takes whole rows (grid
// stride); lane l holds chunks l, l + 64, ... of its row, all loads in flight
// at once.  The row's max / min is a wave butterfly (values only: the
// forward parameters need no index); LET's 1/s and delta are staged in LDS
// once per workgroup.  Same operation order as the per-block kernel below.
template <typename TX, int CH>
__global__ __launch_bounds__(NT) void act_fwd_row_kernel(
    const TX* __restrict__ X, int64_t T, int64_t C, int bits, const float* __restrict__ s,
    const float* __restrict__ delta, TX* __restrict__ xdq, uint8_t* __restrict__ codes,
    float* __restrict__ hout, float* __restrict__ zout) {
  // LET only: 1/s then delta, as float4 slots [k][half][lane] so that one
  // 128-bit LDS read per (k, half) covers 1 KiB of consecutive LDS.
  extern __shared__ float4 shl4[];
  constexpr int SLOTS = CH * 128;
  const bool let = s || delta;
  const int nch = int(C / 8);
  if (let) {
    for (int i = threadIdx.x; i < SLOTS; i += NT) {
      const int64_t c0 = 8 * int64_t((i & 63) + 64 * (i >> 7)) + 4 * ((i >> 6) & 1);
      float a[4], b[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t c = c0 + q;
        a[q] = (s && c < C) ? div_rn(1.0f, s[c]) : 1.0f;
        b[q] = (delta && c < C) ? delta[c] : 0.0f;
      }
      shl4[i] = make_float4(a[0], a[1], a[2], a[3]);
      shl4[SLOTS + i] = make_float4(b[0], b[1], b[2], b[3]);
    }
    __syncthreads();
  }
  const int lane = threadIdx.x & 63;
  const int64_t nw = int64_t(gridDim.x) * (NT / 64);
  const bool quant = bits < 16;
  const float qmax = quant ? float((1 << bits) - 1) : 0.0f;
  // rows of up to 8 chunks per lane: the wave's next row is loaded while this
  // one is reduced and quantised
  constexpr bool PF = CH <= 8;
  Chunk8<TX> nxt[PF ? CH : 1];
  const int64_t row0 = int64_t(blockIdx.x) * (NT / 64) + (threadIdx.x >> 6);
  if constexpr (PF) {
    if (row0 < T) {
#pragma unroll
      for (int k = 0; k < CH; ++k) {
        const int j = lane + 64 * k;
        if (j < nch) nxt[k].load(X + row0 * C + 8 * j);
      }
    }
  }
  for (int64_t row = row0; row < T; row += nw) {
    const TX* xr = X + row * C;
    Chunk8<TX> raw[CH];
    if constexpr (PF) {
#pragma unroll
      for (int k = 0; k < CH; ++k) raw[k] = nxt[k];
      if (row + nw < T) {
#pragma unroll
        for (int k = 0; k < CH; ++k) {
          const int j = lane + 64 * k;
          if (j < nch) nxt[k].load(X + (row + nw) * C + 8 * j);
        }
      }
    } else {
#pragma unroll
      for (int k = 0; k < CH; ++k) {
        const int j = lane + 64 * k;
        if (j < nch) raw[k].load(xr + 8 * j);
      }
    }
    // x~ = (x - delta) (1/s), one rounding per operation
    auto xt8 = [&](int k, float (&o)[8]) {
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = raw[k].at(e);
      if (!let) return;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float4 r = shl4[(2 * k + h) * 64 + lane];
        const float4 d = shl4[SLOTS + (2 * k + h) * 64 + lane];
        o[4 * h + 0] = (o[4 * h + 0] - d.x) * r.x;
        o[4 * h + 1] = (o[4 * h + 1] - d.y) * r.y;
        o[4 * h + 2] = (o[4 * h + 2] - d.z) * r.z;
        o[4 * h + 3] = (o[4 * h + 3] - d.w) * r.w;
      }
    };
    if (!quant) {
#pragma unroll
      for (int k = 0; k < CH; ++k) {
        const int j = lane + 64 * k;
        if (j >= nch) continue;
        float d[8];
        xt8(k, d);
        store8(xdq + row * C + 8 * j, d);
      }
      continue;
    }
    float mx = -FLT_MAX, mn = FLT_MAX;
#pragma unroll
    for (int k = 0; k < CH; ++k) {
      if (lane + 64 * k >= nch) continue;
      float v[8];
      xt8(k, v);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        mx = fmaxf(mx, v[e]);
        mn = fminf(mn, v[e]);
      }
    }
    mx = wave_max(mx);
    mn = wave_min(mn);
    const QParams p = make_qparams(mx, mn, 1.0f, 1.0f, qmax);
    const float lo = -p.z, hi = qmax - p.z;     // clamp as one med3 (exact integers)
    // x~ is recomputed from the packed row (and LDS) rather than kept as
    // fp32 from the range pass: the opaque register and memory barrier
    // stops the compiler from holding every converted value live
    asm volatile("" ::: "memory");
#pragma unroll
    for (int k = 0; k < CH; ++k)
#pragma unroll
      for (int i = 0; i < Chunk8<TX>::NV; ++i)
        asm volatile("" : "+v"(raw[k].v[i].x), "+v"(raw[k].v[i].y), "+v"(raw[k].v[i].z),
                     "+v"(raw[k].v[i].w));
#pragma unroll
    for (int k = 0; k < CH; ++k) {
      const int j = lane + 64 * k;
      if (j >= nch) continue;
      float v[8], q[8], d[8];
      xt8(k, v);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float tq = __builtin_amdgcn_fmed3f(rintf(v[e] * p.r), lo, hi);
        d[e] = tq * p.h;
        q[e] = tq + p.z;
      }
      if (xdq) store8(xdq + row * C + 8 * j, d);
      if (codes) store8_codes(codes + row * C + 8 * j, q);
    }
    if (lane == 0) {
      if (hout) hout[row] = p.h;
      if (zout) zout[row] = p.z;
    }
  }
}

// ------------------------------------------------------------------ LWC forward, wave per row
// Whole-row groups (group = c_in, up to 512 * CH weights): each wave takes
// whole rows (grid stride), lane l holding chunks l, l + 64, ... as loaded.
// LET's s is staged in LDS once per workgroup as float4 slots [k][half][lane]
// (conflict-free 128-bit reads).  Same Eq. 2 arithmetic as lwc_fwd_kernel:
// the clamp is a median of three on rint(u) (q - z stays an exact integer).
template <typename TW, typename TQ, int CH, bool CODES>
__global__ __launch_bounds__(NT) void lwc_fwd_row_kernel(
    const TW* __restrict__ W, int64_t c_out, int64_t c_in, const float* __restrict__ s,
    const float* __restrict__ gl, const float* __restrict__ bl, int bits, TQ* __restrict__ wdq,
    uint8_t* __restrict__ codes, float* __restrict__ hout, float* __restrict__ zout) {
  extern __shared__ float4 shw4[];
  constexpr int SLOTS = CH * 128;
  const int nch = int(c_in / 8);
  if (s) {
    for (int i = threadIdx.x; i < SLOTS; i += NT) {
      const int64_t c0 = 8 * int64_t((i & 63) + 64 * (i >> 7)) + 4 * ((i >> 6) & 1);
      float a[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) a[q] = c0 + q < c_in ? s[c0 + q] : 1.0f;
      shw4[i] = make_float4(a[0], a[1], a[2], a[3]);
    }
    __syncthreads();
  }
  const int lane = threadIdx.x & 63;
  const int64_t nw = int64_t(gridDim.x) * (NT / 64);
  const float qmax = float((1 << bits) - 1);
  for (int64_t row = int64_t(blockIdx.x) * (NT / 64) + (threadIdx.x >> 6); row < c_out;
       row += nw) {
    const TW* wr = W + row * c_in;
    Chunk8<TW> raw[CH];
#pragma unroll
    for (int k = 0; k < CH; ++k) {
      const int j = lane + 64 * k;
      if (j < nch) raw[k].load(wr + 8 * j);
    }
    // w~ = w * s, one rounding
    auto wt8 = [&](int k, float (&o)[8]) {
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = raw[k].at(e);
      if (!s) return;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float4 m = shw4[(2 * k + h) * 64 + lane];
        o[4 * h + 0] *= m.x;
        o[4 * h + 1] *= m.y;
        o[4 * h + 2] *= m.z;
        o[4 * h + 3] *= m.w;
      }
    };
    float mx = -FLT_MAX, mn = FLT_MAX;
#pragma unroll
    for (int k = 0; k < CH; ++k) {
      if (lane + 64 * k >= nch) continue;
      float v[8];
      wt8(k, v);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        mx = fmaxf(mx, v[e]);
        mn = fminf(mn, v[e]);
      }
    }
    mx = wave_max(mx);
    mn = wave_min(mn);
    const QParams p = make_qparams(mx, mn, clip_strength(gl[row]), clip_strength(bl[row]), qmax);
    const float lo = -p.z, hi = qmax - p.z;
    // recompute w~ from the packed row rather than hold it in fp32
    asm volatile("" ::: "memory");
#pragma unroll
    for (int k = 0; k < CH; ++k)
#pragma unroll
      for (int i = 0; i < Chunk8<TW>::NV; ++i)
        asm volatile("" : "+v"(raw[k].v[i].x), "+v"(raw[k].v[i].y), "+v"(raw[k].v[i].z),
                     "+v"(raw[k].v[i].w));
#pragma unroll
    for (int k = 0; k < CH; ++k) {
      const int j = lane + 64 * k;
      if (j >= nch) continue;
      float v[8], d[8], q[8];
      wt8(k, v);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float tq = __builtin_amdgcn_fmed3f(rintf(v[e] * p.r), lo, hi);
        d[e] = tq * p.h;
        q[e] = tq + p.z;
      }
      if (wdq) store8(wdq + row * c_in + 8 * j, d);
      if constexpr (CODES) store8_codes(codes + row * c_in + 8 * j, q);
    }
    if (lane == 0) {
      if (hout) hout[row] = p.h;
      if (zout) zout[row] = p.z;
    }
  }
}

// ------------------------------------------------------------------ activation forward
// x~ = (x - delta) * (1/s); per token row Eq. 2 with gamma = beta = 1.
template <typename TX, typename TQ, int KC, int NTB = NT>
__global__ __launch_bounds__(NTB) void act_fwd_kernel(
    const TX* __restrict__ X, int64_t T, int64_t C, int bits, const float* __restrict__ s,
    const float* __restrict__ delta, int R, TQ* __restrict__ xdq, uint8_t* __restrict__ codes,
    float* __restrict__ hout, float* __restrict__ zout, bool sym) {
  __shared__ MinMax shm[NTB / 64];
  const int tid = threadIdx.x;
  const int cpr = int(C / 8);
  const bool quant = bits < 16;
  const float qmax = quant ? float((1 << bits) - 1) : 0.0f;
  const float qs = quant ? float((1 << (bits - 1)) - 1) : 0.0f;
  float rs[KC][8], dl[KC][8];
#pragma unroll
  for (int k = 0; k < KC; ++k) {
    const int j = tid + NTB * k;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      rs[k][e] = 1.0f;
      dl[k][e] = 0.0f;
    }
    if (j < cpr) {
      if (s) {
        load8(s + 8 * j, rs[k]);
#pragma unroll
        for (int e = 0; e < 8; ++e) rs[k][e] = div_rn(1.0f, rs[k][e]);
      }
      if (delta) load8(delta + 8 * j, dl[k]);
    }
  }
  const bool let = s || delta;
  const int64_t r0 = int64_t(blockIdx.x) * R;
  const int64_t r1 = min(T, r0 + R);
  for (int64_t row = r0; row < r1; ++row) {
    float v[KC][8];
    MinMax st = minmax_init();
#pragma unroll
    for (int k = 0; k < KC; ++k) {
      const int j = tid + NTB * k;
      if (j < cpr) {
        load8(X + row * C + 8 * j, v[k]);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          if (let) v[k][e] = (v[k][e] - dl[k][e]) * rs[k][e];
          minmax_add(st, v[k][e], 8 * j + e);
        }
      }
    }
    if (!quant) {
#pragma unroll
      for (int k = 0; k < KC; ++k) {
        const int j = tid + NTB * k;
        if (j < cpr && xdq) store8(xdq + row * C + 8 * j, v[k]);
      }
      continue;
    }
    st = block_minmax<NTB>(st, shm);
    int iab;
    float sgn;
    const QParams p = sym ? make_sym_qparams(st.mx, st.imx, st.mn, st.imn, qs, iab, sgn)
                          : make_qparams(st.mx, st.mn, 1.0f, 1.0f, qmax);
#pragma unroll
    for (int k = 0; k < KC; ++k) {
      const int j = tid + NTB * k;
      if (j < cpr) {
        float q[8], d[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          q[e] = quant_elem(v[k][e], p, qmax).q;
          d[e] = dequant(q[e], p);
        }
        if (xdq) store8(xdq + row * C + 8 * j, d);
        if (codes) store8_codes(codes + row * C + 8 * j, q);
      }
    }
    if (tid == 0) {
      if (hout) hout[row] = p.h;
      if (zout) zout[row] = p.z;
    }
  }
}

// ------------------------------------------------------------------ activation backward
// dx~ per element (straight-through with the row scale's gradient); per column
// partial sums over this block's rows of dx~ * x~ and of dx~.
// One barrier per block reduction (lds_barrier): the LDS slots of the two
// reductions alternate, and a wave reads each slot before it arrives at the
// other reduction's barrier, so no second barrier guards the rewrite.
template <typename TX, int KC, int NTB = NT>
__global__ __launch_bounds__(NTB) void act_bwd_kernel(
    const TX* __restrict__ X, int64_t T, int64_t C, int bits, const float* __restrict__ s,
    const float* __restrict__ delta, int R, const float* __restrict__ dXdq,
    float* __restrict__ dXt, float* __restrict__ p_sx, float* __restrict__ p_s1, bool sym) {
  __shared__ MinMax shm[NTB / 64];
  __shared__ float2 shs[NTB / 64];
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int cpr = int(C / 8);
  const bool quant = bits < 16;
  const float qmax = quant ? float((1 << bits) - 1) : 0.0f;
  const float qs = quant ? float((1 << (bits - 1)) - 1) : 0.0f;
  float rs[KC][8], dl[KC][8], asx[KC][8], as1[KC][8];
#pragma unroll
  for (int k = 0; k < KC; ++k) {
    const int j = tid + NTB * k;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      rs[k][e] = 1.0f;
      dl[k][e] = 0.0f;
      asx[k][e] = 0.0f;
      as1[k][e] = 0.0f;
    }
    if (j < cpr) {
      if (s) {
        load8(s + 8 * j, rs[k]);
#pragma unroll
        for (int e = 0; e < 8; ++e) rs[k][e] = div_rn(1.0f, rs[k][e]);
      }
      if (delta) load8(delta + 8 * j, dl[k]);
    }
  }
  const bool let = s || delta;
  const int64_t r0 = int64_t(blockIdx.x) * R;
  const int64_t r1 = min(T, r0 + R);
  // up to two chunks per thread, the next row's X and dX^ are loaded while
  // this row is reduced (wider rows would spill)
  constexpr bool PF = KC <= 2;
  Chunk8<TX> xn[KC];
  float gn[KC][8];
  auto issue = [&](int64_t row) {
#pragma unroll
    for (int k = 0; k < KC; ++k) {
      const int j = tid + NTB * k;
      if (j < cpr) {
        xn[k].load(X + row * C + 8 * j);
        load8(dXdq + row * C + 8 * j, gn[k]);
      }
    }
  };
  if constexpr (PF) {
    if (r0 < r1) issue(r0);
  }
  for (int64_t row = r0; row < r1; ++row) {
    float v[KC][8], g[KC][8];
    MinMax st = minmax_init();
    if constexpr (PF) {
#pragma unroll
      for (int k = 0; k < KC; ++k) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          v[k][e] = xn[k].at(e);
          g[k][e] = gn[k][e];
        }
      }
      if (row + 1 < r1) issue(row + 1);
    } else {
#pragma unroll
      for (int k = 0; k < KC; ++k) {
        const int j = tid + NTB * k;
        if (j < cpr) {
          load8(X + row * C + 8 * j, v[k]);
          load8(dXdq + row * C + 8 * j, g[k]);
        }
      }
    }
#pragma unroll
    for (int k = 0; k < KC; ++k) {
      const int j = tid + NTB * k;
      if (j < cpr) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          if (let) v[k][e] = (v[k][e] - dl[k][e]) * rs[k][e];
          minmax_add(st, v[k][e], 8 * j + e);
        }
      }
    }
    if (quant) {
      wave_minmax(st.mx, st.imx, st.mn, st.imn);
      if ((tid & 63) == 0) shm[wave] = st;
      lds_barrier();
      st = shm[0];
#pragma unroll
      for (int w = 1; w < NTB / 64; ++w) {
        sel_max(st.mx, st.imx, shm[w].mx, shm[w].imx);
        sel_min(st.mn, st.imn, shm[w].mn, shm[w].imn);
      }
      int iab = -1;
      float sgn = 1.0f;
      const QParams p = sym ? make_sym_qparams(st.mx, st.imx, st.mn, st.imn, qs, iab, sgn)
                            : make_qparams(st.mx, st.mn, 1.0f, 1.0f, qmax);
      float2 sums = make_float2(0.f, 0.f);
      bool mk[KC][8];
#pragma unroll
      for (int k = 0; k < KC; ++k) {
        const int j = tid + NTB * k;
        if (j < cpr) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const QElem qe = quant_elem(v[k][e], p, qmax);
            mk[k][e] = qe.m;
            const float t = qe.q - p.z;
            const float th = qe.m ? t - qe.u : t;
            sums.x += g[k][e] * th;
            sums.y += qe.m ? 0.0f : g[k][e];
          }
        }
      }
      sums.x = wave_sum(sums.x);
      sums.y = wave_sum(sums.y);
      if ((tid & 63) == 0) shs[wave] = sums;
      lds_barrier();
      sums = shs[0];
#pragma unroll
      for (int w = 1; w < NTB / 64; ++w) {
        sums.x += shs[w].x;
        sums.y += shs[w].y;
      }
      const QGrad qg = quant_group_grad(sums.x, sums.y, st.mx, st.mn, p, qmax);
      // symmetric: the zero point is fixed, dh = S_h goes to the absmax
      // element through |x|max = qs * h, with that element's sign
      const float dab = sym ? (p.hclamp ? 0.0f : sgn * div_rn(sums.x, qs)) : 0.0f;
#pragma unroll
      for (int k = 0; k < KC; ++k) {
        const int j = tid + NTB * k;
        if (j < cpr) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int col = 8 * j + e;
            float x = mk[k][e] ? g[k][e] : 0.0f;
            if (sym) {
              if (col == iab) x += dab;
            } else {
              if (col == st.imx) x += qg.dmx;
              if (col == st.imn) x += qg.dmn;
            }
            g[k][e] = x;
          }
        }
      }
    }
#pragma unroll
    for (int k = 0; k < KC; ++k) {
      const int j = tid + NTB * k;
      if (j < cpr) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          asx[k][e] += g[k][e] * v[k][e];
          as1[k][e] += g[k][e];
        }
        if (dXt) store8(dXt + row * C + 8 * j, g[k]);
      }
    }
  }
#pragma unroll
  for (int k = 0; k < KC; ++k) {
    const int j = tid + NTB * k;
    if (j < cpr) {
      if (p_sx) store8(p_sx + int64_t(blockIdx.x) * C + 8 * j, asx[k]);
      if (p_s1) store8(p_s1 + int64_t(blockIdx.x) * C + 8 * j, as1[k]);
    }
  }
}

// ------------------------------------------------------------------ quantiser initialisation
// One wave per group: the group's (max, min) of w~ = s (.) w, and from them
// the MinMax starting point of a quantiser variant: PACT (hi, lo) = (max,
// min); LSQ (h, z) = Eq. 2's step and zero point at clip strength 1; LWC
// keeps its logits at 4 (clip strength sigmoid(4)).
template <typename TW>
__global__ __launch_bounds__(NT) void wquant_init_kernel(const TW* __restrict__ W, int64_t n_groups,
                                                         int64_t c_in, int group,
                                                         const float* __restrict__ s, int bits,
                                                         int quant, float* __restrict__ p1,
                                                         float* __restrict__ p2) {
  const int lane = threadIdx.x & 63;
  const int64_t gi = int64_t(blockIdx.x) * (NT / 64) + (threadIdx.x >> 6);
  if (gi >= n_groups) return;
  const int64_t ng = c_in / group;
  const int64_t row = gi / ng, c0 = (gi % ng) * group;
  float mx = -FLT_MAX, mn = FLT_MAX;
  int imx = INT_MAX, imn = INT_MAX;
  for (int i = lane; i < group; i += 64) {
    float w = load1(W + row * c_in + c0 + i);
    if (s) w = w * s[c0 + i];
    sel_max(mx, imx, w, i);
    sel_min(mn, imn, w, i);
  }
  wave_minmax(mx, imx, mn, imn);
  if (lane != 0) return;
  const float qmax = float((1 << bits) - 1);
  if (quant == WQ_PACT) {
    p1[gi] = mx;
    p2[gi] = mn;
  } else if (quant == WQ_LSQ) {
    const QParams p = make_qparams(mx, mn, 1.0f, 1.0f, qmax);
    p1[gi] = p.h;
    p2[gi] = p.z;
  } else {
    p1[gi] = 4.0f;
    p2[gi] = 4.0f;
  }
}

int kc_for(int64_t cols) {
  const int64_t need = (cols / 8 + NT - 1) / NT;
  if (need <= 1) return 1;
  if (need <= 2) return 2;
  if (need <= 4) return 4;
  if (need <= 8) return 8;
  if (need <= 16) return 16;
  return 0;
}

// Blocks of `threads` threads (with lds bytes of dynamic LDS each) that the current
// device keeps resident at once: compute units times the kernel's occupancy,
// cached per (kernel, LDS bytes, device).
int resident_blocks(const void* kernel, size_t lds = 0, int threads = NT) {
  struct Entry { const void* k; size_t lds; int dev, n; };
  static std::mutex mu;
  static std::vector<Entry> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) dev = 0;
  {
    std::lock_guard<std::mutex> g(mu);
    for (const Entry& e : cache)
      if (e.k == kernel && e.lds == lds && e.dev == dev) return e.n;
  }
  int cus = 0, per = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kernel, threads, lds) != hipSuccess)
    return 1024;
  const int n = std::max(1, cus * per);
  std::lock_guard<std::mutex> g(mu);
  cache.push_back(Entry{kernel, lds, dev, n});
  return n;
}

int rows_per_block(int64_t rows, int64_t target_blocks) {
  return int(std::max<int64_t>(1, (rows + target_blocks - 1) / target_blocks));
}

constexpr int64_t LWC_BLOCKS = 768;
constexpr int64_t ACT_BLOCKS = 768;

#define OQ_KC_SWITCH(KCV, ...)                      \
  switch (KCV) {                                    \
    case 1: { constexpr int KC = 1; __VA_ARGS__; } break;  \
    case 2: { constexpr int KC = 2; __VA_ARGS__; } break;  \
    case 4: { constexpr int KC = 4; __VA_ARGS__; } break;  \
    case 8: { constexpr int KC = 8; __VA_ARGS__; } break;  \
    case 16: { constexpr int KC = 16; __VA_ARGS__; } break; \
    default: return hipErrorInvalidValue;           \
  }

bool small_group(int64_t group) {
  return group >= 8 && group <= 512 && (group & (group - 1)) == 0;
}

}  // namespace

bool quant_shape_supported(int64_t c_in, int64_t group) {
  if (c_in <= 0 || c_in % 8 || group <= 0 || c_in % group) return false;
  if (kc_for(c_in) == 0) return false;
  return small_group(group) || group == c_in;
}

hipError_t lwc_fwd(const void* W, bool w_bf16, int64_t c_out, int64_t c_in, const float* s,
                   const float* gl, const float* bl, int bits, int64_t group, void* W_dq,
                   bool dq_bf16, uint8_t* codes, float* h, float* z, hipStream_t st,
                   float4* gstat, int quant) {
  if (!quant_shape_supported(c_in, group)) return hipErrorInvalidValue;
  if (c_out <= 0) return hipSuccess;
  if (gstat && (s || !small_group(group) || quant != WQ_LWC)) return hipErrorInvalidValue;
  if (quant < WQ_LWC || quant > WQ_LSQ) return hipErrorInvalidValue;
  if (small_group(group) && !s && quant == WQ_LWC) {
    const int64_t nchunk = c_out * c_in / 8;
    const int64_t waves = std::min<int64_t>((nchunk + 511) / 512, 256 * 32);
    const dim3 grid(unsigned((waves * 64 + NT - 1) / NT));
    auto go = [&](auto tw, auto tq, auto gc) {
      using TW = decltype(tw);
      using TQ = decltype(tq);
      constexpr int Gc = decltype(gc)::value;
      if (codes)
        hipLaunchKernelGGL((lwc_fwd_coal_kernel<TW, TQ, Gc, true>), grid, dim3(NT), 0, st,
                           static_cast<const TW*>(W), nchunk, gl, bl, bits, static_cast<TQ*>(W_dq),
                           codes, h, z, gstat);
      else
        hipLaunchKernelGGL((lwc_fwd_coal_kernel<TW, TQ, Gc, false>), grid, dim3(NT), 0, st,
                           static_cast<const TW*>(W), nchunk, gl, bl, bits, static_cast<TQ*>(W_dq),
                           codes, h, z, gstat);
    };
    auto by_g = [&](auto tw, auto tq) {
      switch (group / 8) {
        case 1: go(tw, tq, std::integral_constant<int, 1>{}); break;
        case 2: go(tw, tq, std::integral_constant<int, 2>{}); break;
        case 4: go(tw, tq, std::integral_constant<int, 4>{}); break;
        case 8: go(tw, tq, std::integral_constant<int, 8>{}); break;
        case 16: go(tw, tq, std::integral_constant<int, 16>{}); break;
        case 32: go(tw, tq, std::integral_constant<int, 32>{}); break;
        default: go(tw, tq, std::integral_constant<int, 64>{}); break;
      }
    };
    if (w_bf16) dq_bf16 ? by_g(uint16_t{}, uint16_t{}) : by_g(uint16_t{}, float{});
    else dq_bf16 ? by_g(float{}, uint16_t{}) : by_g(float{}, float{});
    return hipGetLastError();
  }
  const int64_t per_lane = (c_in / 8 + 63) / 64;
  if (group == c_in && per_lane <= 32 && quant == WQ_LWC) {
    const int ch = per_lane <= 2 ? 2 : per_lane <= 4 ? 4 : per_lane <= 8 ? 8 : per_lane <= 12 ? 12
                 : per_lane <= 16 ? 16 : per_lane <= 24 ? 24 : 32;
    const unsigned lds = s ? unsigned(ch) * 128u * 16u : 0u;
    // one round of resident workgroups, each wave looping over rows
    const int64_t want = (c_out + NT / 64 - 1) / (NT / 64);
    auto run = [&](auto tw, auto tq, auto chc) {
      using TW = decltype(tw);
      using TQ = decltype(tq);
      constexpr int CHc = decltype(chc)::value;
      if (codes) {
        auto* k = lwc_fwd_row_kernel<TW, TQ, CHc, true>;
        const dim3 grid(unsigned(std::min<int64_t>(want, resident_blocks((const void*)k, lds))));
        hipLaunchKernelGGL(k, grid, dim3(NT), lds, st, static_cast<const TW*>(W), c_out, c_in, s,
                           gl, bl, bits, static_cast<TQ*>(W_dq), codes, h, z);
      } else {
        auto* k = lwc_fwd_row_kernel<TW, TQ, CHc, false>;
        const dim3 grid(unsigned(std::min<int64_t>(want, resident_blocks((const void*)k, lds))));
        hipLaunchKernelGGL(k, grid, dim3(NT), lds, st, static_cast<const TW*>(W), c_out, c_in, s,
                           gl, bl, bits, static_cast<TQ*>(W_dq), codes, h, z);
      }
    };
    auto by_ch = [&](auto tw, auto tq) {
      switch (ch) {
        case 2: run(tw, tq, std::integral_constant<int, 2>{}); break;
        case 4: run(tw, tq, std::integral_constant<int, 4>{}); break;
        case 8: run(tw, tq, std::integral_constant<int, 8>{}); break;
        case 12: run(tw, tq, std::integral_constant<int, 12>{}); break;
        case 16: run(tw, tq, std::integral_constant<int, 16>{}); break;
        case 24: run(tw, tq, std::integral_constant<int, 24>{}); break;
        default: run(tw, tq, std::integral_constant<int, 32>{}); break;
      }
    };
    if (w_bf16) dq_bf16 ? by_ch(uint16_t{}, uint16_t{}) : by_ch(uint16_t{}, float{});
    else dq_bf16 ? by_ch(float{}, uint16_t{}) : by_ch(float{}, float{});
    return hipGetLastError();
  }
  const int R = rows_per_block(c_out, LWC_BLOCKS);
  const dim3 grid(unsigned((c_out + R - 1) / R));
  const bool whole = !small_group(group);
  const int kc = kc_for(c_in);
  auto go = [&](auto tw, auto tq, auto kcc, auto wr) {
    using TW = decltype(tw);
    using TQ = decltype(tq);
    constexpr int KCc = decltype(kcc)::value;
    constexpr bool WR = decltype(wr)::value;
    hipLaunchKernelGGL((lwc_fwd_kernel<TW, TQ, KCc, WR>), grid, dim3(NT), 0, st,
                       static_cast<const TW*>(W), c_out, c_in, s, gl, bl, bits, int(group), R,
                       static_cast<TQ*>(W_dq), codes, h, z, quant);
  };
  auto by_kc = [&](auto tw, auto tq, auto wr) -> hipError_t {
    OQ_KC_SWITCH(kc, go(tw, tq, std::integral_constant<int, KC>{}, wr))
    return hipSuccess;
  };
  auto by_wr = [&](auto tw, auto tq) -> hipError_t {
    return whole ? by_kc(tw, tq, std::true_type{}) : by_kc(tw, tq, std::false_type{});
  };
  hipError_t e;
  if (w_bf16) e = dq_bf16 ? by_wr(uint16_t{}, uint16_t{}) : by_wr(uint16_t{}, float{});
  else e = dq_bf16 ? by_wr(float{}, uint16_t{}) : by_wr(float{}, float{});
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

hipError_t wquant_init(const void* W, bool w_bf16, int64_t c_out, int64_t c_in, const float* s,
                       int bits, int64_t group, int quant, float* p1, float* p2, hipStream_t st) {
  if (group <= 0 || c_in % group || quant < WQ_LWC || quant > WQ_LSQ) return hipErrorInvalidValue;
  const int64_t n = c_out * (c_in / group);
  if (n <= 0) return hipSuccess;
  const dim3 grid(unsigned((n + NT / 64 - 1) / (NT / 64)));
  if (w_bf16)
    hipLaunchKernelGGL(wquant_init_kernel<uint16_t>, grid, dim3(NT), 0, st,
                       static_cast<const uint16_t*>(W), n, c_in, int(group), s, bits, quant, p1, p2);
  else
    hipLaunchKernelGGL(wquant_init_kernel<float>, grid, dim3(NT), 0, st,
                       static_cast<const float*>(W), n, c_in, int(group), s, bits, quant, p1, p2);
  return hipGetLastError();
}

int64_t lwc_bwd_nparts(int64_t c_out) {
  if (c_out <= 0) return 0;
  const int R = rows_per_block(c_out, LWC_BLOCKS);
  return (c_out + R - 1) / R;
}

bool lwc_bwd_sums_parts(int64_t c_out, int64_t c_in, int64_t group, bool has_s, bool want_ds) {
  return quant_shape_supported(c_in, group) && small_group(group) && !has_s && !want_ds &&
         c_out * c_in < (int64_t(1) << 34);
}

hipError_t lwc_bwd(const void* W, bool w_bf16, int64_t c_out, int64_t c_in, const float* s,
                   const float* gl, const float* bl, int bits, int64_t group, const float* dW,
                   float* dgl, float* dbl, float* dW_tilde, float* ds_parts, hipStream_t st,
                   int parts, int64_t part_stride, int quant) {
  if (!quant_shape_supported(c_in, group)) return hipErrorInvalidValue;
  if (c_out <= 0) return hipSuccess;
  if (quant < WQ_LWC || quant > WQ_LSQ || (quant != WQ_LWC && parts != 1))
    return hipErrorInvalidValue;
  if (parts < 1 || (parts > 1 && (!lwc_bwd_sums_parts(c_out, c_in, group, s, ds_parts) ||
                                  part_stride < c_out * c_in || part_stride % 4)))
    return hipErrorInvalidValue;
  // LSQ's gradient scale 1/sqrt(n * Q_P), n = weights per step size
  const float gs = float(1.0 / std::sqrt(double(group) * double((1 << bits) - 1)));
  if (quant == WQ_LWC && lwc_bwd_sums_parts(c_out, c_in, group, s, ds_parts)) {
    const int E = int(std::min<int64_t>(group, 32));
    const int64_t nrun = c_out * (c_in / E);
    const dim3 grid(unsigned((nrun + NT - 1) / NT));
    auto run = [&](auto tw, auto ec) {
      using TW = decltype(tw);
      constexpr int Ec = decltype(ec)::value;
      if (dW_tilde)
        hipLaunchKernelGGL((lwc_bwd_run_kernel<TW, Ec, true>), grid, dim3(NT), 0, st,
                           static_cast<const TW*>(W), c_out, c_in, gl, bl, bits, int(group), dW,
                           dgl, dbl, dW_tilde, parts, part_stride);
      else
        hipLaunchKernelGGL((lwc_bwd_run_kernel<TW, Ec, false>), grid, dim3(NT), 0, st,
                           static_cast<const TW*>(W), c_out, c_in, gl, bl, bits, int(group), dW,
                           dgl, dbl, dW_tilde, parts, part_stride);
    };
    auto by_e = [&](auto tw) {
      switch (E) {
        case 8: run(tw, std::integral_constant<int, 8>{}); break;
        case 16: run(tw, std::integral_constant<int, 16>{}); break;
        case 32: run(tw, std::integral_constant<int, 32>{}); break;
        default: run(tw, std::integral_constant<int, 64>{}); break;
      }
    };
    if (w_bf16) by_e(uint16_t{});
    else by_e(float{});
    return hipGetLastError();
  }
  const bool whole = !small_group(group);
  const int kc = kc_for(c_in);
  auto go = [&](auto tw, auto kcc, auto wr) {
    using TW = decltype(tw);
    constexpr int KC0 = decltype(kcc)::value;
    constexpr bool WR = decltype(wr)::value;
    // whole rows of more than two chunks per thread (wider than 4,096):
    // 512-thread blocks, half the chunks per thread (11,008-wide rows
    // measured 247 -> 173 us; 4,096-wide ones are faster at 256 threads)
    constexpr int NTc = WR && KC0 >= 4 ? 512 : NT;
    constexpr int KCc = NTc == 512 ? KC0 / 2 : KC0;
    if (s || ds_parts) {
      // the ds partials are one row per block: the block count is the fixed
      // lwc_bwd_nparts(c_out) the workspace was sized for
      const int R = rows_per_block(c_out, LWC_BLOCKS);
      hipLaunchKernelGGL((lwc_bwd_kernel<TW, KCc, WR, true, NTc>), dim3(unsigned((c_out + R - 1) / R)),
                         dim3(NTc), 0, st, static_cast<const TW*>(W), c_out, c_in, s, gl, bl, bits,
                         int(group), R, dW, dgl, dbl, dW_tilde, ds_parts, quant, gs);
    } else {
      // no partials: one round of resident blocks
      const int R = rows_per_block(
          c_out, resident_blocks(reinterpret_cast<const void*>(lwc_bwd_kernel<TW, KCc, WR, false, NTc>),
                                 0, NTc));
      hipLaunchKernelGGL((lwc_bwd_kernel<TW, KCc, WR, false, NTc>), dim3(unsigned((c_out + R - 1) / R)),
                         dim3(NTc), 0, st, static_cast<const TW*>(W), c_out, c_in, s, gl, bl, bits,
                         int(group), R, dW, dgl, dbl, dW_tilde, ds_parts, quant, gs);
    }
  };
  auto by_kc = [&](auto tw, auto wr) -> hipError_t {
    OQ_KC_SWITCH(kc, go(tw, std::integral_constant<int, KC>{}, wr))
    return hipSuccess;
  };
  auto by_wr = [&](auto tw) -> hipError_t {
    return whole ? by_kc(tw, std::true_type{}) : by_kc(tw, std::false_type{});
  };
  hipError_t e = w_bf16 ? by_wr(uint16_t{}) : by_wr(float{});
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

hipError_t act_fwd(const void* X, bool x_bf16, int64_t T, int64_t C, int bits, const float* s,
                   const float* delta, void* X_dq, bool dq_bf16, uint8_t* codes, float* h,
                   float* z, hipStream_t st, bool sym) {
  const int kc = kc_for(C);
  if (C <= 0 || C % 8 || kc == 0) return hipErrorInvalidValue;
  if (T <= 0) return hipSuccess;
  if (sym && bits >= 16) sym = false;
  const int64_t per_lane = (C / 8 + 63) / 64;
  if (x_bf16 == dq_bf16 && per_lane <= 32 && (X_dq || bits < 16) && !sym) {
    const int ch = per_lane <= 2 ? 2 : per_lane <= 4 ? 4 : per_lane <= 8 ? 8 : per_lane <= 12 ? 12
                 : per_lane <= 16 ? 16 : per_lane <= 24 ? 24 : 32;
    const unsigned lds = (s || delta) ? unsigned(ch) * 128u * 2u * 16u : 0u;
    // up to 2048 workgroups, each wave looping over rows (one round of the
    // resident count measured 3-9% slower for 4096-channel rows with LET)
    const dim3 grid(unsigned(std::min<int64_t>((T + NT / 64 - 1) / (NT / 64), 2048)));
    auto run = [&](auto tx, auto chc) {
      using TX = decltype(tx);
      constexpr int CHc = decltype(chc)::value;
      hipLaunchKernelGGL((act_fwd_row_kernel<TX, CHc>), grid, dim3(NT), lds, st,
                         static_cast<const TX*>(X), T, C, bits, s, delta, static_cast<TX*>(X_dq),
                         codes, h, z);
    };
    auto by_ch = [&](auto tx) {
      switch (ch) {
        case 2: run(tx, std::integral_constant<int, 2>{}); break;
        case 4: run(tx, std::integral_constant<int, 4>{}); break;
        case 8: run(tx, std::integral_constant<int, 8>{}); break;
        case 12: run(tx, std::integral_constant<int, 12>{}); break;
        case 16: run(tx, std::integral_constant<int, 16>{}); break;
        case 24: run(tx, std::integral_constant<int, 24>{}); break;
        default: run(tx, std::integral_constant<int, 32>{}); break;
      }
    };
    if (x_bf16) by_ch(uint16_t{});
    else by_ch(float{});
    return hipGetLastError();
  }
  const int R = rows_per_block(T, ACT_BLOCKS);
  const dim3 grid(unsigned((T + R - 1) / R));
  auto go = [&](auto tx, auto tq, auto kcc) {
    using TX = decltype(tx);
    using TQ = decltype(tq);
    constexpr int KCc = decltype(kcc)::value;
    if constexpr (KCc >= 8) {
      // wide rows: twice the threads per row, half the chunks per thread
      hipLaunchKernelGGL((act_fwd_kernel<TX, TQ, KCc / 2, 2 * NT>), grid, dim3(2 * NT), 0, st,
                         static_cast<const TX*>(X), T, C, bits, s, delta, R, static_cast<TQ*>(X_dq),
                         codes, h, z, sym);
    } else {
      hipLaunchKernelGGL((act_fwd_kernel<TX, TQ, KCc>), grid, dim3(NT), 0, st,
                         static_cast<const TX*>(X), T, C, bits, s, delta, R, static_cast<TQ*>(X_dq),
                         codes, h, z, sym);
    }
  };
  auto by_kc = [&](auto tx, auto tq) -> hipError_t {
    OQ_KC_SWITCH(kc, go(tx, tq, std::integral_constant<int, KC>{}))
    return hipSuccess;
  };
  hipError_t e;
  if (x_bf16) e = dq_bf16 ? by_kc(uint16_t{}, uint16_t{}) : by_kc(uint16_t{}, float{});
  else e = dq_bf16 ? by_kc(float{}, uint16_t{}) : by_kc(float{}, float{});
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

int64_t act_bwd_nparts(int64_t T) {
  if (T <= 0) return 0;
  const int R = rows_per_block(T, ACT_BLOCKS);
  return (T + R - 1) / R;
}

hipError_t act_bwd(const void* X, bool x_bf16, int64_t T, int64_t C, int bits, const float* s,
                   const float* delta, const float* dXdq, float* dXt, float* p_sx, float* p_s1,
                   hipStream_t st, bool sym) {
  const int kc = kc_for(C);
  if (C <= 0 || C % 8 || kc == 0) return hipErrorInvalidValue;
  if (T <= 0) return hipSuccess;
  const int R = rows_per_block(T, ACT_BLOCKS);
  const dim3 grid(unsigned((T + R - 1) / R));
  auto go = [&](auto tx, auto kcc) {
    using TX = decltype(tx);
    constexpr int KCc = decltype(kcc)::value;
    if constexpr (KCc >= 8) {
      // wide rows: twice the threads per row, half the chunks per thread
      // (256 threads with 8 chunks each leave one wave per SIMD)
      hipLaunchKernelGGL((act_bwd_kernel<TX, KCc / 2, 2 * NT>), grid, dim3(2 * NT), 0, st,
                         static_cast<const TX*>(X), T, C, bits, s, delta, R, dXdq, dXt, p_sx, p_s1,
                         sym && bits < 16);
    } else {
      hipLaunchKernelGGL((act_bwd_kernel<TX, KCc>), grid, dim3(NT), 0, st,
                         static_cast<const TX*>(X), T, C, bits, s, delta, R, dXdq, dXt, p_sx, p_s1,
                         sym && bits < 16);
    }
  };
  auto by_kc = [&](auto tx) -> hipError_t {
    OQ_KC_SWITCH(kc, go(tx, std::integral_constant<int, KC>{}))
    return hipSuccess;
  };
  hipError_t e = x_bf16 ? by_kc(uint16_t{}) : by_kc(float{});
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

}  // namespace oq
