// Deployment of the calibrated weights (Sec. 4.5, Table "tab:speed"): the
// integer codes W_q of Eq.2 stored as low-bit strings, and the weight-only
// quantised linear Y = X W^T + B that reads them, with W = (W_q - z) * h per
// group (Eq.2's dequantisation) and 16-bit activations.
//
// Storage: each output row's codes form one little-endian bit string (code j
// at bits j*bits .. j*bits + bits - 1), rows back to back.  Because c_in is a
// multiple of 32, every run of 32 codes is exactly `bits` whole dwords: the
// unit a lane loads.
//
// The linear is a batched GEMV and HBM-bound at decode batch sizes: every
// packed weight byte is read once, the few activation rows sit in LDS.  A code
// is widened without a conversion instruction: OR-ing it into the mantissa of
// the bf16 value 128.0 gives exactly 128 + q (bf16 holds the integers up to
// 256), and one v_dot2 multiplies two such codes with two activations.  With
// p = sum x (128 + q) over a 32-code run and xs = sum x over the same run,
// that run contributes h * (p - (128 + z) * xs).
#include <algorithm>
#include <mutex>
#include <vector>

#include "common.h"
#include "packed.h"

namespace oq {
namespace {

constexpr int PACK_THREADS = 256;
constexpr int PL_THREADS = 256;               // 4 waves
constexpr int PL_WAVES = PL_THREADS / 64;
constexpr int PL_ROWS = 2;                    // output rows a wave works on together
constexpr int PL_U = 2;                       // runs per lane loaded together
constexpr uint32_t BF16_128_PAIR = 0x43004300u;
constexpr size_t PL_LDS_MAX = 160 * 1024;
constexpr int64_t PM_MIN_TOKENS = 8;          // batches from this size run on matrix cores

typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));

// ------------------------------------------------------------------ packing
// One thread per run of 32 codes: 32 input bytes -> BITS output dwords.  Only
// the low BITS bits of each code are stored.
template <int BITS>
__global__ __launch_bounds__(PACK_THREADS) void pack_codes_kernel(const uint8_t* __restrict__ codes,
                                                                  int64_t n_runs,
                                                                  uint32_t* __restrict__ out) {
  const int64_t stride = int64_t(gridDim.x) * PACK_THREADS;
  for (int64_t i = int64_t(blockIdx.x) * PACK_THREADS + threadIdx.x; i < n_runs; i += stride) {
    const uint4* src = reinterpret_cast<const uint4*>(codes + 32 * i);
    const uint4 a = src[0], b = src[1];
    const uint32_t w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    uint32_t o[BITS];
#pragma unroll
    for (int k = 0; k < BITS; ++k) o[k] = 0;
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      const uint32_t c = (w[j >> 2] >> (8 * (j & 3))) & ((1u << BITS) - 1);
      const int pos = j * BITS;
      o[pos >> 5] |= c << (pos & 31);
      if ((pos & 31) + BITS > 32) o[(pos >> 5) + 1] |= c >> (32 - (pos & 31));
    }
    uint32_t* dst = out + i * BITS;
#pragma unroll
    for (int k = 0; k < BITS; ++k) dst[k] = o[k];
  }
}

// ------------------------------------------------------------------ pair order
// A run's 32 codes are consumed as 16 pairs.  For 4- and 2-bit codes a pair is
// two fields 16 bits apart in one dword, so one AND/OR extracts both; other
// widths pair neighbours.  The activation row is staged in LDS in the same
// pair order: pair p multiplies activations pair_lo(p) (low half) and
// pair_hi(p) (high half) of the run.
template <int BITS>
OQ_DEV constexpr int pair_lo(int p) {
  return BITS == 4 ? 8 * (p >> 2) + (p & 3) : BITS == 2 ? 16 * (p >> 3) + (p & 7) : 2 * p;
}
template <int BITS>
OQ_DEV constexpr int pair_hi(int p) {
  return BITS == 4 ? pair_lo<BITS>(p) + 4 : BITS == 2 ? pair_lo<BITS>(p) + 8 : 2 * p + 1;
}

// bits pos .. pos + BITS - 1 of the run's string (pos known at compile time)
template <int BITS>
OQ_DEV uint32_t field(const uint32_t* w, int pos) {
  const int d = pos >> 5, o = pos & 31;
  uint32_t v = w[d] >> o;
  if (o + BITS > 32) v |= w[d + 1] << (32 - o);
  return v & ((1u << BITS) - 1);
}

// (a & mask) | magic in one instruction.  The compiler emits an AND and an OR
// here: both constants are literals, and a gfx9 three-operand instruction
// takes no literal, so they are passed in registers.
OQ_DEV uint32_t and_or(uint32_t a, uint32_t mask, uint32_t magic) {
  uint32_t r;
  asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(mask), "v"(magic));
  return r;
}

// The 16 pairs of bf16 values (128 + q_lo, 128 + q_hi) of one run.
template <int BITS>
OQ_DEV void code_pairs(const uint32_t* w, uint32_t* p, uint32_t mask, uint32_t magic) {
  if constexpr (BITS == 4) {
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int i = 0; i < 4; ++i) p[4 * d + i] = and_or(w[d] >> (4 * i), mask, magic);
  } else if constexpr (BITS == 2) {
#pragma unroll
    for (int d = 0; d < 2; ++d)
#pragma unroll
      for (int i = 0; i < 8; ++i) p[8 * d + i] = and_or(w[d] >> (2 * i), mask, magic);
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i)
      p[i] = field<BITS>(w, 2 * i * BITS) | (field<BITS>(w, (2 * i + 1) * BITS) << 16) | BF16_128_PAIR;
  }
}

OQ_DEV float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_v, a),
                                         __builtin_bit_cast(bf16x2_v, b), c, false);
}

template <int BITS>
OQ_DEV void load_run(const uint32_t* __restrict__ src, uint32_t* w) {
  if constexpr (BITS == 4) {
    const uint4 v = *reinterpret_cast<const uint4*>(src);
    w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
  } else if constexpr (BITS == 2) {
    const uint2 v = *reinterpret_cast<const uint2*>(src);
    w[0] = v.x; w[1] = v.y;
  } else {
#pragma unroll
    for (int k = 0; k < BITS; ++k) w[k] = src[k];
  }
}

// ------------------------------------------------------------------ the linear
// LDS: for token t and run k, the 16 activation pairs as four 16-byte quads at
// xq[(t * 4 + quad) * nrun + k] (consecutive lanes read consecutive quads),
// then the run sums xs[t * nrun + k].
//
// Waves take groups of PL_ROWS output rows in turn.  A wave walks its work as
// blocks of PL_U runs per lane (lane l of k-block b holds runs
// 64 * (b * PL_U + u) + l) and loads block j + 1 before it computes block j,
// so the next loads are always in flight; the first block is loaded before the
// activations are staged.  At the last k-block of a row group the wave sums
// its lanes and stores the group's outputs.  Rows past c_out (the last group)
// re-read row c_out - 1 and store nothing.
template <int BITS, int NT>
__global__ __launch_bounds__(PL_THREADS) void packed_linear_kernel(
    const uint16_t* __restrict__ X, int n_tok, int64_t c_in, const uint32_t* __restrict__ P,
    int runs_per_group, int group_shift, const float* __restrict__ H, const float* __restrict__ Z,
    const float* __restrict__ bias, int64_t c_out, void* __restrict__ Y, bool y_bf16) {
  extern __shared__ uint4 lds_q[];
  const int nrun = int(c_in / 32);
  float* xs_l = reinterpret_cast<float*>(lds_q + size_t(NT) * 4 * nrun);
  const int lane = threadIdx.x & 63;
  const int64_t nwave = int64_t(gridDim.x) * PL_WAVES;
  const int ng = nrun / runs_per_group;
  const int row_dw = nrun * BITS;
  const int nkb = (nrun + 64 * PL_U - 1) / (64 * PL_U);
  // the two fields of a pair in one dword (4- and 2-bit codes) and the bf16 128.0 pair
  const uint32_t pair_mask = BITS == 4 ? 0x000F000Fu : 0x00030003u;
  const uint32_t magic = BF16_128_PAIR;

  // the group of run k (runs_per_group a power of two: a shift)
  auto group_of = [&](int k) {
    return group_shift >= 0 ? (k >> group_shift) : int(unsigned(k) / unsigned(runs_per_group));
  };
  // Load k-block kb of row group rg (first row rg * PL_ROWS < c_out).
  auto issue = [&](int64_t rg, int kb, uint32_t (&w)[PL_U][PL_ROWS][BITS], float (&hh)[PL_U][PL_ROWS],
                   float (&zz)[PL_U][PL_ROWS]) {
    const uint32_t* prow[PL_ROWS];
    const float *hrow[PL_ROWS], *zrow[PL_ROWS];
#pragma unroll
    for (int r = 0; r < PL_ROWS; ++r) {
      const int64_t row = std::min<int64_t>(rg * PL_ROWS + r, c_out - 1);
      prow[r] = P + row * row_dw;
      hrow[r] = H + row * ng;
      zrow[r] = Z + row * ng;
    }
#pragma unroll
    for (int u = 0; u < PL_U; ++u) {
      const int k = 64 * (kb * PL_U + u) + lane;
      if (k < nrun) {
        const int g = group_of(k);
#pragma unroll
        for (int r = 0; r < PL_ROWS; ++r) {
          load_run<BITS>(prow[r] + k * BITS, w[u][r]);
          hh[u][r] = hrow[r][g];
          zz[u][r] = zrow[r][g];
        }
      }
    }
  };

  float acc[PL_ROWS][NT];
#pragma unroll
  for (int r = 0; r < PL_ROWS; ++r)
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[r][t] = 0.f;

  // Compute k-block kb of row group rg from its loaded block; at the last
  // k-block sum the lanes and store the group's outputs.
  auto compute = [&](int64_t rg, int kb, const uint32_t (&w)[PL_U][PL_ROWS][BITS],
                     const float (&hh)[PL_U][PL_ROWS], const float (&zz)[PL_U][PL_ROWS]) {
#pragma unroll
    for (int u = 0; u < PL_U; ++u) {
      const int k = 64 * (kb * PL_U + u) + lane;
      if (k < nrun) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const uint4* xq = lds_q + size_t(t) * 4 * nrun + k;
          uint32_t xp[16];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const uint4 v = xq[size_t(q) * nrun];
            xp[4 * q] = v.x; xp[4 * q + 1] = v.y; xp[4 * q + 2] = v.z; xp[4 * q + 3] = v.w;
          }
          const float xs = xs_l[t * nrun + k];
#pragma unroll
          for (int r = 0; r < PL_ROWS; ++r) {
            uint32_t cp[16];
            code_pairs<BITS>(w[u][r], cp, pair_mask, magic);
            float p = 0.f;
#pragma unroll
            for (int m = 0; m < 16; ++m) p = dot2_bf16(xp[m], cp[m], p);
            acc[r][t] = __builtin_fmaf(hh[u][r], __builtin_fmaf(-(128.f + zz[u][r]), xs, p), acc[r][t]);
          }
        }
      }
    }
    if (kb == nkb - 1) {
#pragma unroll
      for (int r = 0; r < PL_ROWS; ++r) {
        const int64_t row = rg * PL_ROWS + r;
        const float b = (bias != nullptr && row < c_out) ? bias[row] : 0.f;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const float v = wave_sum(acc[r][t]) + b;
          acc[r][t] = 0.f;
          if (lane == 0 && row < c_out && t < n_tok) {
            if (y_bf16)
              static_cast<uint16_t*>(Y)[int64_t(t) * c_out + row] = f2bf(v);
            else
              static_cast<float*>(Y)[int64_t(t) * c_out + row] = v;
          }
        }
      }
    }
  };

  // the wave's blocks in order: row groups wave, wave + nwave, ..., each
  // with k-blocks 0 .. nkb - 1
  int64_t rg = int64_t(blockIdx.x) * PL_WAVES + (threadIdx.x >> 6);
  int kb = 0;
  uint32_t wa[PL_U][PL_ROWS][BITS], wb[PL_U][PL_ROWS][BITS];
  float ha[PL_U][PL_ROWS], za[PL_U][PL_ROWS], hb[PL_U][PL_ROWS], zb[PL_U][PL_ROWS];
  const bool any = rg * PL_ROWS < c_out;
  if (any) issue(rg, kb, wa, ha, za);

  // stage the activation rows: one thread per (token, run)
  for (int idx = threadIdx.x; idx < NT * nrun; idx += PL_THREADS) {
    const int t = idx / nrun, k = idx - t * nrun;
    uint32_t u[16];
    if (t < n_tok) {
      const uint4* src = reinterpret_cast<const uint4*>(X + int64_t(t) * c_in + 32 * int64_t(k));
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint4 v = src[e];
        u[4 * e] = v.x; u[4 * e + 1] = v.y; u[4 * e + 2] = v.z; u[4 * e + 3] = v.w;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 16; ++e) u[e] = 0;
    }
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 32; ++j) s += bf2f(uint16_t(u[j >> 1] >> (16 * (j & 1))));
    uint32_t pr[16];
#pragma unroll
    for (int p = 0; p < 16; ++p) {
      const int a = pair_lo<BITS>(p), b = pair_hi<BITS>(p);
      const uint32_t xa = (u[a >> 1] >> (16 * (a & 1))) & 0xffffu;
      const uint32_t xb = (u[b >> 1] >> (16 * (b & 1))) & 0xffffu;
      pr[p] = xa | (xb << 16);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q)
      lds_q[(size_t(t) * 4 + q) * nrun + k] = make_uint4(pr[4 * q], pr[4 * q + 1], pr[4 * q + 2], pr[4 * q + 3]);
    xs_l[t * nrun + k] = s;
  }
  __syncthreads();
  if (!any) return;

  // two load buffers in turn: the next block loads while this one computes
  while (true) {
    int64_t rg2 = kb + 1 < nkb ? rg : rg + nwave;
    int kb2 = kb + 1 < nkb ? kb + 1 : 0;
    bool more = rg2 * PL_ROWS < c_out;
    if (more) issue(rg2, kb2, wb, hb, zb);
    compute(rg, kb, wa, ha, za);
    if (!more) break;
    rg = rg2;
    kb = kb2;
    rg2 = kb + 1 < nkb ? rg : rg + nwave;
    kb2 = kb + 1 < nkb ? kb + 1 : 0;
    more = rg2 * PL_ROWS < c_out;
    if (more) issue(rg2, kb2, wa, ha, za);
    compute(rg, kb, wb, hb, zb);
    if (!more) break;
    rg = rg2;
    kb = kb2;
  }
}

size_t linear_lds(int nt, int64_t c_in) { return size_t(nt) * size_t(c_in / 32) * (64 + 4); }

// Workgroups of the kernel that the current device keeps resident at once,
// cached per (kernel, LDS bytes, device).
int resident(const void* kernel, size_t lds) {
  struct Entry { const void* k; size_t lds; int dev, n; };
  static std::mutex mu;
  static std::vector<Entry> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) dev = 0;
  std::lock_guard<std::mutex> g(mu);
  for (const Entry& e : cache)
    if (e.k == kernel && e.lds == lds && e.dev == dev) return e.n;
  int cus = 0, per = 0;
  if (hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, int(PL_LDS_MAX)) !=
          hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kernel, PL_THREADS, lds) != hipSuccess)
    return 256;
  const int n = std::max(1, cus * per);
  cache.push_back(Entry{kernel, lds, dev, n});
  return n;
}

// Lets the kernel take up to PL_LDS_MAX bytes of dynamic LDS on the current
// device (once per kernel and device).
hipError_t allow_lds(const void* kernel) {
  struct Entry { const void* k; int dev; };
  static std::mutex mu;
  static std::vector<Entry> done;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> g(mu);
  for (const Entry& d : done)
    if (d.k == kernel && d.dev == dev) return hipSuccess;
  e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, int(PL_LDS_MAX));
  if (e == hipSuccess) done.push_back(Entry{kernel, dev});
  return e;
}

// ------------------------------------------------------------------ the linear on matrix cores
// For batches of 8 or more tokens and groups of 128 codes.  A workgroup owns
// 16 output rows (or two tiles of 16, RT = 2); its eight waves take the rows'
// groups g = wave, wave + 8, ...
// For group g a lane (f, i) (f = lane / 16, i = lane % 16) loads run 4 g + f
// of row i (BITS dwords); matrix instruction m (0..3) of the group multiplies
// codes 8 m .. 8 m + 7 of each lane's run, widened to 128 + q in bf16 (exact),
// with the activations of the same columns, 32 (4 g + f) + 8 m + e, as its B
// operand: the group's p = sum x (128 + q) for 16 rows x 16 tokens, fp32.  The
// lanes also sum those activations (xs = sum x), and the group adds
// h (p - (128 + z) xs) to each output, in fp32, as in the VALU kernel.  The
// eight waves' partial outputs are added in fixed order through LDS.
//
// Activations reach the B operand through LDS: each wave copies a group's
// 16-token x 128-channel block (4 KiB) with four global_load_lds_dwordx4, one
// instruction per four tokens, so every instruction reads four whole 256-byte
// token rows (a 16-lane B operand read straight from global memory would touch
// sixteen rows 8 KiB apart).  In LDS token t's 16-byte chunk c sits in slot
// c ^ t of the token's 256 bytes, so the lanes of one fragment read hit
// distinct banks.  Each wave double-buffers its blocks: the copies of group
// g + 8 are in flight while group g computes.
constexpr int PM_THREADS = 512;                // 8 waves share a tile's groups
constexpr int PM_WAVES = PM_THREADS / 64;
constexpr int PM_GROUP = 128;
constexpr int64_t PM_RT2_ROWS = 16384;         // output rows from which a workgroup takes 32

// 16 bytes per lane, global -> LDS (lane l's bytes land at LDS byte address
// lds + 16 l); inline assembly, so the kernel waits for it (vmcnt) itself.
// m0 (the copy's LDS base) is saved and restored around it, with one wait
// state between its write and the copy that reads it.
OQ_DEV void copy16_lds(const void* g, uint32_t lds) {
  const uint32_t m0v = __builtin_amdgcn_readfirstlane(lds);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(m0v), "v"(g)
      : "memory");
}
OQ_DEV void wait_vm0() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
OQ_DEV uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>(
      (__attribute__((address_space(3))) const char*)(p)));
}

// dynamic LDS of the kernel: h and z of the workgroup's 16 rt rows, then two
// activation blocks per wave and 16-token block, of tpb staged tokens each
// (the partial-output exchange reuses them)
size_t mfma_lds(int rt, int ntb, int tpb, int64_t c_in) {
  return size_t(2 * 16 * rt) * size_t(c_in / PM_GROUP) * sizeof(float) +
         size_t(PM_WAVES) * 2 * size_t(ntb) * size_t(tpb) * PM_GROUP * 2;
}

// NTB blocks of 16 tokens; TPB = 8 stages only the first 8 tokens of the
// block (batches of at most 8: half the LDS, so more workgroups per CU).  RT
// tiles of 16 rows per workgroup: each activation fragment read from LDS
// feeds RT matrix instructions.  A row's arithmetic does not depend on RT.
template <int BITS, int NTB, int TPB, int RT>
__global__ __launch_bounds__(PM_THREADS) void packed_mfma_kernel(
    const uint16_t* __restrict__ X, int n_tok, int64_t c_in, const uint32_t* __restrict__ packed,
    const float* __restrict__ h, const float* __restrict__ z, const float* __restrict__ bias,
    int64_t c_out, void* __restrict__ Y, bool y_bf16) {
  static_assert(TPB == 16 || (TPB == 8 && NTB == 1), "staged tokens per block");
  constexpr int XBLK = TPB * PM_GROUP * 2;     // bytes of one group's block
  constexpr int XB = NTB * XBLK;               // one wave's buffer: a group's NTB blocks
  extern __shared__ float lds[];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int f = lane >> 4, i = lane & 15;
  const int64_t o0 = int64_t(blockIdx.x) * 16 * RT;
  const int ng = int(c_in / PM_GROUP);
  const int64_t runs_row = c_in / 32;
  float* hz = lds;                             // [2][16 RT][ng]: h, then 128 + z
  char* xbuf = reinterpret_cast<char*>(lds + 32 * RT * ng) + size_t(wave) * 2 * XB;
  // this lane's A rows (rows past c_out re-read the last row and store nothing)
  const uint32_t* prow[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
    prow[rt] = packed + min(o0 + 16 * rt + i, c_out - 1) * runs_row * BITS;

  // copies of group g's activations into buffer b: instruction j of block tb
  // carries tokens 16 tb + 4 j .. + 3 (lane l: token 4 j + l / 16 of the
  // block, slot l % 16 holding chunk (l % 16) ^ token).  Instructions whose
  // tokens all lie past n_tok are skipped; single tokens past it read the
  // last token: they only feed accumulator columns that are never stored.
  auto stage = [&](int g, int b) {
#pragma unroll
    for (int tb = 0; tb < NTB; ++tb)
#pragma unroll
      for (int j = 0; j < TPB / 4; ++j) {
        const int t0 = 16 * tb + 4 * j;
        if (t0 < n_tok) {
          const int tt = 4 * j + (lane >> 4);
          const int t = min(16 * tb + tt, n_tok - 1);
          const int c = (lane & 15) ^ tt;
          copy16_lds(X + int64_t(t) * c_in + PM_GROUP * int64_t(g) + 8 * c,
                     lds_addr(xbuf + b * XB + tb * XBLK + j * 1024));
        }
      }
  };
  uint32_t wn[RT][BITS];
  if (wave < ng) {
    stage(wave, 0);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) load_run<BITS>(prow[rt] + (4 * int64_t(wave) + f) * BITS, wn[rt]);
  }
  {
    const int64_t nrow = min<int64_t>(16 * RT, c_out - o0);
    for (int e = tid; e < 16 * RT * ng; e += PM_THREADS) {
      const int64_t src = (o0 + min<int64_t>(e / ng, nrow - 1)) * ng + e % ng;
      hz[e] = h[src];
      hz[16 * RT * ng + e] = 128.0f + z[src];
    }
  }
  __syncthreads();
  f32x4_t y[RT][NTB];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int tb = 0; tb < NTB; ++tb) y[rt][tb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  int b = 0;
  for (int g = wave; g < ng; g += PM_WAVES, b ^= 1) {
    // group g's copies and codes, issued one turn ago, have landed
    wait_vm0();
    uint32_t w[RT][BITS];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int k = 0; k < BITS; ++k) w[rt][k] = wn[rt][k];
    if (g + PM_WAVES < ng) {
      stage(g + PM_WAVES, b ^ 1);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
        load_run<BITS>(prow[rt] + (4 * int64_t(g + PM_WAVES) + f) * BITS, wn[rt]);
    }
    float hr[RT][4], zr[RT][4];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        hr[rt][r] = hz[(16 * rt + 4 * f + r) * ng + g];
        zr[rt][r] = hz[16 * RT * ng + (16 * rt + 4 * f + r) * ng + g];
      }
    f32x4_t acc[RT][NTB];
    float xs[NTB];
#pragma unroll
    for (int tb = 0; tb < NTB; ++tb) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) acc[rt][tb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      xs[tb] = 0.f;
    }
    // columns past the staged tokens (TPB = 8) re-read tokens 0..7: never stored
    const int ti = i & (TPB - 1);
    const char* xb = xbuf + b * XB + ti * 256;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      bf16x8_t av[RT];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        uint32_t a[4];
#pragma unroll
        for (int p = 0; p < 4; ++p)
          a[p] = field<BITS>(w[rt], (8 * m + 2 * p) * BITS) |
                 (field<BITS>(w[rt], (8 * m + 2 * p + 1) * BITS) << 16) | BF16_128_PAIR;
        av[rt] = __builtin_bit_cast(bf16x8_t, make_uint4(a[0], a[1], a[2], a[3]));
      }
#pragma unroll
      for (int tb = 0; tb < NTB; ++tb) {
        const uint4 xv =
            *reinterpret_cast<const uint4*>(xb + tb * XBLK + 16 * ((4 * f + m) ^ ti));
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
          acc[rt][tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              av[rt], __builtin_bit_cast(bf16x8_t, xv), acc[rt][tb], 0, 0, 0);
        xs[tb] = dot2_bf16(xv.x, 0x3f803f80u, xs[tb]);
        xs[tb] = dot2_bf16(xv.y, 0x3f803f80u, xs[tb]);
        xs[tb] = dot2_bf16(xv.z, 0x3f803f80u, xs[tb]);
        xs[tb] = dot2_bf16(xv.w, 0x3f803f80u, xs[tb]);
      }
    }
#pragma unroll
    for (int tb = 0; tb < NTB; ++tb) {
      // xs of token 16 tb + i over the whole group: the four lanes f of column i
      float s = xs[tb];
      s += __shfl_xor(s, 16);
      s += __shfl_xor(s, 32);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int r = 0; r < 4; ++r) y[rt][tb][r] += hr[rt][r] * (acc[rt][tb][r] - zr[rt][r] * s);
    }
  }
  // every wave's copies have landed (each waited before its last group), so
  // the activation buffers can hold the partial outputs: lane (f, i) holds
  // rows 16 rt + 4 f + r of the workgroup for token 16 tb + i
  __syncthreads();
  float* red = lds + 32 * RT * ng;             // [PM_WAVES][RT][NTB * 16][17]
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int tb = 0; tb < NTB; ++tb)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        red[((wave * RT + rt) * NTB * 16 + 16 * tb + i) * 17 + 4 * f + r] = y[rt][tb][r];
  __syncthreads();
  for (int e = tid; e < RT * NTB * 16 * 16; e += PM_THREADS) {
    const int rr = e % 16, t = (e / 16) % (NTB * 16), rt = e / (16 * NTB * 16);
    const int64_t o = o0 + 16 * rt + rr;
    if (t < n_tok && o < c_out) {
      float v = red[(rt * NTB * 16 + t) * 17 + rr];
#pragma unroll
      for (int w8 = 1; w8 < PM_WAVES; ++w8) v += red[((w8 * RT + rt) * NTB * 16 + t) * 17 + rr];
      if (bias) v += bias[o];
      if (y_bf16) static_cast<uint16_t*>(Y)[int64_t(t) * c_out + o] = f2bf(v);
      else static_cast<float*>(Y)[int64_t(t) * c_out + o] = v;
    }
  }
}

template <int BITS, int NTB, int TPB, int RT>
hipError_t launch_mfma_rt(const uint16_t* X, int n_tok, int64_t c_in, const uint8_t* packed,
                          const float* h, const float* z, const float* bias, int64_t c_out, void* Y,
                          bool y_bf16, hipStream_t stream) {
  auto k = packed_mfma_kernel<BITS, NTB, TPB, RT>;
  const size_t lds = mfma_lds(RT, NTB, TPB, c_in);
  if (lds > 64 * 1024) {
    const hipError_t e = allow_lds(reinterpret_cast<const void*>(k));
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k, dim3(unsigned((c_out + 16 * RT - 1) / (16 * RT))), dim3(PM_THREADS), lds,
                     stream, X, n_tok, c_in, reinterpret_cast<const uint32_t*>(packed), h, z, bias,
                     c_out, Y, y_bf16);
  return hipGetLastError();
}

template <int BITS, int NTB, int TPB>
hipError_t launch_mfma(int rt, const uint16_t* X, int n_tok, int64_t c_in, const uint8_t* packed,
                       const float* h, const float* z, const float* bias, int64_t c_out, void* Y,
                       bool y_bf16, hipStream_t stream) {
  if (rt == 2)
    return launch_mfma_rt<BITS, NTB, TPB, 2>(X, n_tok, c_in, packed, h, z, bias, c_out, Y, y_bf16, stream);
  return launch_mfma_rt<BITS, NTB, TPB, 1>(X, n_tok, c_in, packed, h, z, bias, c_out, Y, y_bf16, stream);
}

template <int BITS, int NT>
hipError_t launch_linear(const uint16_t* X, int n_tok, int64_t c_in, const uint8_t* packed,
                         int64_t group, const float* h, const float* z, const float* bias,
                         int64_t c_out, void* Y, bool y_bf16, hipStream_t stream) {
  auto k = packed_linear_kernel<BITS, NT>;
  const size_t lds = linear_lds(NT, c_in);
  const int64_t want = (c_out + PL_WAVES * PL_ROWS - 1) / (PL_WAVES * PL_ROWS);
  const int64_t blocks = std::min<int64_t>(want, resident(reinterpret_cast<const void*>(k), lds));
  const int rpg = int(group / 32);
  const int shift = (rpg & (rpg - 1)) == 0 ? __builtin_ctz(unsigned(rpg)) : -1;
  hipLaunchKernelGGL(k, dim3(unsigned(blocks)), dim3(PL_THREADS), lds, stream, X, n_tok, c_in,
                     reinterpret_cast<const uint32_t*>(packed), rpg, shift, h, z, bias, c_out, Y, y_bf16);
  return hipGetLastError();
}

template <int BITS>
hipError_t linear_bits(const uint16_t* X, int64_t n_tok, int64_t c_in, const uint8_t* packed,
                       int64_t group, const float* h, const float* z, const float* bias,
                       int64_t c_out, void* Y, bool y_bf16, hipStream_t stream) {
  const size_t es = y_bf16 ? 2 : 4;
  if (n_tok >= PM_MIN_TOKENS && group == PM_GROUP) {
    // matrix cores: launches of up to 32 tokens, or 16 where two blocks
    // of 32 tokens exceed LDS; batches of at most 8 stage 8 tokens per group
    const int most = mfma_lds(1, 2, 16, c_in) <= PL_LDS_MAX ? 32 : 16;
    for (int64_t t0 = 0; t0 < n_tok;) {
      const int take = int(std::min<int64_t>(n_tok - t0, most));
      const uint16_t* x = X + t0 * c_in;
      void* y = static_cast<char*>(Y) + size_t(t0) * size_t(c_out) * es;
      // two row tiles per workgroup from 16384 rows, and from 8192 rows for
      // two token blocks, where LDS allows (a row's sums do not depend on it)
      const int ntb = take > 16 ? 2 : 1, tpb = take > 8 ? 16 : 8;
      const bool two = c_out >= PM_RT2_ROWS || (c_out >= PM_RT2_ROWS / 2 && ntb == 2);
      const int rt = two && mfma_lds(2, ntb, tpb, c_in) <= PL_LDS_MAX ? 2 : 1;
      const hipError_t e =
          take <= 8    ? launch_mfma<BITS, 1, 8>(rt, x, take, c_in, packed, h, z, bias, c_out, y, y_bf16, stream)
          : take <= 16 ? launch_mfma<BITS, 1, 16>(rt, x, take, c_in, packed, h, z, bias, c_out, y, y_bf16, stream)
                       : launch_mfma<BITS, 2, 16>(rt, x, take, c_in, packed, h, z, bias, c_out, y, y_bf16, stream);
      if (e != hipSuccess) return e;
      t0 += take;
    }
    return hipSuccess;
  }
  for (int64_t t0 = 0; t0 < n_tok;) {
    const int64_t rem = n_tok - t0;
    int nt = rem >= 8 ? 8 : rem >= 4 ? (rem == 4 ? 4 : 8) : rem >= 2 ? (rem == 2 ? 2 : 4) : 1;
    while (nt > 1 && linear_lds(nt, c_in) > PL_LDS_MAX) nt >>= 1;
    const int take = int(std::min<int64_t>(rem, nt));
    const uint16_t* x = X + t0 * c_in;
    void* y = static_cast<char*>(Y) + size_t(t0) * size_t(c_out) * es;
    hipError_t e;
    switch (nt) {
      case 8: e = launch_linear<BITS, 8>(x, take, c_in, packed, group, h, z, bias, c_out, y, y_bf16, stream); break;
      case 4: e = launch_linear<BITS, 4>(x, take, c_in, packed, group, h, z, bias, c_out, y, y_bf16, stream); break;
      case 2: e = launch_linear<BITS, 2>(x, take, c_in, packed, group, h, z, bias, c_out, y, y_bf16, stream); break;
      default: e = launch_linear<BITS, 1>(x, take, c_in, packed, group, h, z, bias, c_out, y, y_bf16, stream); break;
    }
    if (e != hipSuccess) return e;
    t0 += take;
  }
  return hipSuccess;
}

}  // namespace

hipError_t pack_codes(const uint8_t* codes, int64_t c_out, int64_t c_in, int bits, uint8_t* packed,
                      hipStream_t stream) {
  const int64_t n_runs = c_out * (c_in / 32);
  if (n_runs == 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((n_runs + PACK_THREADS - 1) / PACK_THREADS, 4096);
  uint32_t* out = reinterpret_cast<uint32_t*>(packed);
  const dim3 g{unsigned(blocks)}, b{unsigned(PACK_THREADS)};
  switch (bits) {
    case 2: hipLaunchKernelGGL(pack_codes_kernel<2>, g, b, 0, stream, codes, n_runs, out); break;
    case 3: hipLaunchKernelGGL(pack_codes_kernel<3>, g, b, 0, stream, codes, n_runs, out); break;
    case 4: hipLaunchKernelGGL(pack_codes_kernel<4>, g, b, 0, stream, codes, n_runs, out); break;
    case 5: hipLaunchKernelGGL(pack_codes_kernel<5>, g, b, 0, stream, codes, n_runs, out); break;
    case 6: hipLaunchKernelGGL(pack_codes_kernel<6>, g, b, 0, stream, codes, n_runs, out); break;
    case 7: hipLaunchKernelGGL(pack_codes_kernel<7>, g, b, 0, stream, codes, n_runs, out); break;
    case 8: hipLaunchKernelGGL(pack_codes_kernel<8>, g, b, 0, stream, codes, n_runs, out); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t packed_linear(const uint16_t* X, int64_t n_tok, int64_t c_in, const uint8_t* packed,
                         int bits, int64_t group, const float* h, const float* z,
                         const float* bias, int64_t c_out, void* Y, bool y_bf16,
                         hipStream_t stream) {
  if (n_tok == 0 || c_out == 0) return hipSuccess;
  switch (bits) {
    case 2: return linear_bits<2>(X, n_tok, c_in, packed, group, h, z, bias, c_out, Y, y_bf16, stream);
    case 3: return linear_bits<3>(X, n_tok, c_in, packed, group, h, z, bias, c_out, Y, y_bf16, stream);
    case 4: return linear_bits<4>(X, n_tok, c_in, packed, group, h, z, bias, c_out, Y, y_bf16, stream);
    case 5: return linear_bits<5>(X, n_tok, c_in, packed, group, h, z, bias, c_out, Y, y_bf16, stream);
    case 6: return linear_bits<6>(X, n_tok, c_in, packed, group, h, z, bias, c_out, Y, y_bf16, stream);
    case 7: return linear_bits<7>(X, n_tok, c_in, packed, group, h, z, bias, c_out, Y, y_bf16, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace oq
