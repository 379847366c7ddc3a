// Device helpers shared by the liboq kernels (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

// Every named quantity of the quantisers is one IEEE fp32 rounding: never
// fuse a multiply with the following add.
#pragma clang fp contract(off)

#define OQ_DEV __device__ __forceinline__

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// ------------------------------------------------------------------ bf16 <-> fp32
OQ_DEV float bf2f(uint16_t v) { return __uint_as_float(uint32_t(v) << 16); }

// fp32 -> bf16, round to nearest even (gfx950's v_cvt_pk_bf16_f32).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
OQ_DEV uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f)); }
// Two values packed low (a) and high (b) in one dword.
OQ_DEV uint32_t f2bf2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, bf16x2_t));
}

// ------------------------------------------------------------------ 8-wide element access
// A "chunk" is 8 consecutive elements of a row: 16 bytes of bf16 or 32 bytes of fp32.
OQ_DEV void load8(const uint16_t* p, float v[8]) {
  uint4 q = *reinterpret_cast<const uint4*>(p);
  uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    v[2 * e] = __uint_as_float(w[e] << 16);
    v[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
  }
}
OQ_DEV void load8(const float* p, float v[8]) {
  float4 a = *reinterpret_cast<const float4*>(p);
  float4 b = *reinterpret_cast<const float4*>(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
OQ_DEV void store8(uint16_t* p, const float v[8]) {
  uint4 q;
  q.x = f2bf2(v[0], v[1]);
  q.y = f2bf2(v[2], v[3]);
  q.z = f2bf2(v[4], v[5]);
  q.w = f2bf2(v[6], v[7]);
  *reinterpret_cast<uint4*>(p) = q;
}
OQ_DEV void store8(float* p, const float v[8]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
OQ_DEV void store8_codes(uint8_t* p, const float q[8]) {
  uint2 c;
  c.x = uint32_t(q[0]) | (uint32_t(q[1]) << 8) | (uint32_t(q[2]) << 16) | (uint32_t(q[3]) << 24);
  c.y = uint32_t(q[4]) | (uint32_t(q[5]) << 8) | (uint32_t(q[6]) << 16) | (uint32_t(q[7]) << 24);
  *reinterpret_cast<uint2*>(p) = c;
}

OQ_DEV float load1(const uint16_t* p) { return bf2f(*p); }
OQ_DEV float load1(const float* p) { return *p; }
OQ_DEV void store1(uint16_t* p, float v) { *p = f2bf(v); }
OQ_DEV void store1(float* p, float v) { *p = v; }

// ------------------------------------------------------------------ reductions
// (max, lowest index) and (min, lowest index) selections: associative and
// commutative, so any reduction tree gives the same answer.
OQ_DEV void sel_max(float& v, int& i, float ov, int oi) {
  if (ov > v || (ov == v && oi < i)) { v = ov; i = oi; }
}
OQ_DEV void sel_min(float& v, int& i, float ov, int oi) {
  if (ov < v || (ov == v && oi < i)) { v = ov; i = oi; }
}

// Whole-wave reductions on the VALU: DPP exchanges within each 16-lane row
// (quad xor 1, quad xor 2, half-row mirror, row mirror), then the four row
// results read out (lanes 0, 16, 32, 48) and combined in that order.  Every
// lane returns the same value; the order is fixed, so sums are reproducible.
OQ_DEV float dpp_f(float v, int ctrl) {
  switch (ctrl) {
    case 0: return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
    case 1: return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));
    case 2: return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false));
    default: return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, false));
  }
}
OQ_DEV int dpp_i(int v, int ctrl) {
  switch (ctrl) {
    case 0: return __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);
    case 1: return __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);
    case 2: return __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);
    default: return __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false);
  }
}
OQ_DEV float rl_f(float v, int l) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l)); }

OQ_DEV float wave_sum(float v) {
#pragma unroll
  for (int c = 0; c < 4; ++c) v += dpp_f(v, c);
  return ((rl_f(v, 0) + rl_f(v, 16)) + rl_f(v, 32)) + rl_f(v, 48);
}
OQ_DEV float wave_max(float v) {
#pragma unroll
  for (int c = 0; c < 4; ++c) v = fmaxf(v, dpp_f(v, c));
  return fmaxf(fmaxf(rl_f(v, 0), rl_f(v, 16)), fmaxf(rl_f(v, 32), rl_f(v, 48)));
}
OQ_DEV float wave_min(float v) {
#pragma unroll
  for (int c = 0; c < 4; ++c) v = fminf(v, dpp_f(v, c));
  return fminf(fminf(rl_f(v, 0), rl_f(v, 16)), fminf(rl_f(v, 32), rl_f(v, 48)));
}
// max / min with the lowest index among equal values (sel_max / sel_min)
OQ_DEV void wave_minmax(float& mx, int& imx, float& mn, int& imn) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const float omx = dpp_f(mx, c), omn = dpp_f(mn, c);
    const int oimx = dpp_i(imx, c), oimn = dpp_i(imn, c);
    sel_max(mx, imx, omx, oimx);
    sel_min(mn, imn, omn, oimn);
  }
  float rmx = rl_f(mx, 0), rmn = rl_f(mn, 0);
  int rimx = __builtin_amdgcn_readlane(imx, 0), rimn = __builtin_amdgcn_readlane(imn, 0);
#pragma unroll
  for (int l = 16; l < 64; l += 16) {
    sel_max(rmx, rimx, rl_f(mx, l), __builtin_amdgcn_readlane(imx, l));
    sel_min(rmn, rimn, rl_f(mn, l), __builtin_amdgcn_readlane(imn, l));
  }
  mx = rmx; imx = rimx; mn = rmn; imn = rimn;
}

// Butterfly over aligned groups of L lanes (L a power of two <= 64): every
// lane of the group ends with the identical result.
template <int L>
OQ_DEV void group_minmax(float& mx, int& imx, float& mn, int& imn) {
#pragma unroll
  for (int off = 1; off < L; off <<= 1) {
    float omx = __shfl_xor(mx, off);
    int oimx = __shfl_xor(imx, off);
    float omn = __shfl_xor(mn, off);
    int oimn = __shfl_xor(imn, off);
    sel_max(mx, imx, omx, oimx);
    sel_min(mn, imn, omn, oimn);
  }
}
template <int L>
OQ_DEV float group_sum(float v) {
#pragma unroll
  for (int off = 1; off < L; off <<= 1) v += __shfl_xor(v, off);
  return v;
}
OQ_DEV float dyn_group_sum(float v, int L) {
  for (int off = 1; off < L; off <<= 1) v += __shfl_xor(v, off);
  return v;
}
OQ_DEV void dyn_group_minmax(float& mx, int& imx, float& mn, int& imn, int L) {
  for (int off = 1; off < L; off <<= 1) {
    float omx = __shfl_xor(mx, off);
    int oimx = __shfl_xor(imx, off);
    float omn = __shfl_xor(mn, off);
    int oimn = __shfl_xor(imn, off);
    sel_max(mx, imx, omx, oimx);
    sel_min(mn, imn, omn, oimn);
  }
}

// ------------------------------------------------------------------ rounding
// Correctly rounded fp32 quotient and square root whatever the compiler's
// fp32 division / sqrt expansion: one fp64 operation rounded again to fp32
// is the correctly rounded fp32 result (53 >= 2 * 24 + 2 bits).
OQ_DEV float div_rn(float a, float b) { return float(double(a) / double(b)); }
OQ_DEV float sqrt_rn(float a) { return float(__builtin_sqrt(double(a))); }

// ------------------------------------------------------------------ quantiser
// Clip strength: the fp64 sigmoid of the logit, rounded once to fp32.
OQ_DEV float clip_strength(float logit) {
  double t = double(logit);
  return float(1.0 / (1.0 + exp(-t)));
}

struct QParams {
  float gamma, beta, a, b, h, r, z;
  bool hclamp;
};

// Eq. 2 group parameters, fp32 in the fixed order
//   a = gamma*max, b = beta*min, h = (a - b)/qmax, h >= 1e-5, r = 1/h, z = -rint(b*r)
OQ_DEV QParams make_qparams(float mx, float mn, float gamma, float beta, float qmax) {
  QParams p;
  p.gamma = gamma;
  p.beta = beta;
  p.a = gamma * mx;
  p.b = beta * mn;
  float d = p.a - p.b;
  float hr = div_rn(d, qmax);
  p.hclamp = hr < 1e-5f;
  p.h = p.hclamp ? 1e-5f : hr;
  p.r = div_rn(1.0f, p.h);
  p.z = -rintf(p.b * p.r);
  return p;
}

struct QElem {
  float u, q;
  bool m;
};
OQ_DEV QElem quant_elem(float wt, const QParams& p, float qmax) {
  QElem e;
  e.u = wt * p.r;
  float c = rintf(e.u) + p.z;
  e.m = (c >= 0.0f) && (c <= qmax);
  e.q = fminf(fmaxf(c, 0.0f), qmax);
  return e;
}
OQ_DEV float dequant(float q, const QParams& p) { return (q - p.z) * p.h; }

// Straight-through group backward from the sums
//   S_h = sum g*((q - z) - m*u),  S_z = sum g*(1 - m)
struct QGrad {
  float dmx, dmn, dgamma, dbeta;
};
OQ_DEV QGrad quant_group_grad(float s_h, float s_z, float mx, float mn, const QParams& p, float qmax) {
  QGrad g;
  float dh = s_h - s_z * div_rn(p.b, p.h);
  if (p.hclamp) dh = 0.0f;
  float da = div_rn(dh, qmax);
  float db = s_z - da;
  g.dmx = da * p.gamma;
  g.dmn = db * p.beta;
  g.dgamma = da * mx;
  g.dbeta = db * mn;
  return g;
}

// ------------------------------------------------------------------ quantiser variants
// Which weight quantiser fills a group's two parameters p1, p2: LWC's
// clip-strength logits (Eq. 2), PACT's grid thresholds (upper, lower), or
// LSQ's step and zero point (the zero point rounded in the forward).
enum WQuant { WQ_LWC = 0, WQ_PACT = 1, WQ_LSQ = 2 };

OQ_DEV QParams make_group_qparams(int quant, float mx, float mn, float p1, float p2, float qmax) {
  if (quant == WQ_PACT) return make_qparams(p1, p2, 1.0f, 1.0f, qmax);
  if (quant == WQ_LSQ) {
    QParams p;
    p.gamma = p.beta = 1.0f;
    p.a = p.b = 0.0f;
    p.hclamp = p1 < 1e-5f;
    p.h = p.hclamp ? 1e-5f : p1;
    p.r = div_rn(1.0f, p.h);
    p.z = rintf(p2);
    return p;
  }
  return make_qparams(mx, mn, clip_strength(p1), clip_strength(p2), qmax);
}

// One element's share of its group's two backward sums: LWC and LSQ sum
// (S_h, S_z) = (g((q - z) - m u), g(1 - m)); PACT sums the gradient of the
// codes saturated above qmax and below 0.
OQ_DEV void group_terms(int quant, float g, const QElem& qe, const QParams& p, float qmax,
                        float& s1, float& s2) {
  // (selects rather than a branch between the two sums: a reference chosen
  // at run time would put them in scratch memory)
  if (quant == WQ_PACT) {
    s1 += (!qe.m && qe.q == qmax) ? g : 0.0f;
    s2 += (!qe.m && qe.q != qmax) ? g : 0.0f;
    return;
  }
  const float t = qe.q - p.z;
  const float th = qe.m ? t - qe.u : t;
  s1 += g * th;
  s2 += qe.m ? 0.0f : g;
}

// A group's parameter gradients from its two sums, and the max/min
// gradients to route (LWC only: PACT's thresholds and LSQ's step do not
// depend on the weights).  gs is LSQ's gradient scale 1/sqrt(n * qmax).
struct GroupGrad {
  float d1, d2, dmx, dmn;
};
OQ_DEV GroupGrad group_param_grads(int quant, float s1, float s2, float mx, float mn,
                                   const QParams& p, float qmax, float gs) {
  GroupGrad r;
  if (quant == WQ_PACT) {
    r.d1 = s1;
    r.d2 = s2;
    r.dmx = r.dmn = 0.0f;
  } else if (quant == WQ_LSQ) {
    r.d1 = p.hclamp ? 0.0f : gs * s1;
    r.d2 = -(gs * (p.h * s2));
    r.dmx = r.dmn = 0.0f;
  } else {
    const QGrad qg = quant_group_grad(s1, s2, mx, mn, p, qmax);
    r.d1 = qg.dgamma * p.gamma * (1.0f - p.gamma);
    r.d2 = qg.dbeta * p.beta * (1.0f - p.beta);
    r.dmx = qg.dmx;
    r.dmn = qg.dmn;
  }
  return r;
}

// Symmetric per-token absmax quantiser: h = max(|x|max / qs, 1e-5), qs =
// 2^(N-1) - 1, zero point qs + 1.  The absmax element is the lowest index
// holding the largest |x|: from a row's (max, argmax, min, argmin).
OQ_DEV QParams make_sym_qparams(float mx, int imx, float mn, int imn, float qs, int& iab,
                                float& sgn) {
  const float amx = mx, amn = -mn;
  float a;
  if (amx > amn || (amx == amn && imx < imn)) {
    a = amx;
    iab = imx;
    sgn = 1.0f;
  } else {
    a = amn;
    iab = imn;
    sgn = -1.0f;
  }
  QParams p;
  p.gamma = p.beta = 1.0f;
  p.a = a;
  p.b = -a;
  const float hr = div_rn(a, qs);
  p.hclamp = hr < 1e-5f;
  p.h = p.hclamp ? 1e-5f : hr;
  p.r = div_rn(1.0f, p.h);
  p.z = qs + 1.0f;
  return p;
}

