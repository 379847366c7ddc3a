// Matrix products C[M,N] = A[M,K] B[N,K]^T for the calibration step.
//
// bf16 path, K % 64 == 0 (gemm_bf16_w8_kernel): 256x256 output tile per
// workgroup of eight wave64s (two per SIMD), each owning a 128x64 sub-tile as
// 8 x 4 fragments of v_mfma_f32_16x16x32_bf16.  K advances 64 at a time
// through LDS stages (A and B tiles of 256 x 64 bf16 = 32 KiB each; three
// for B and two for A, 160 KiB) filled by global_load_lds_dwordx4 straight
// from global memory.  Fragments are double-buffered in registers per
// 32-wide k-half, and the fragment reads and stage copies are placed by hand
// between groups of four MFMAs: B's copies in one k-half, A's in the other.
// LDS tiles are XOR-swizzled so the lanes of one LDS read hit distinct
// banks; operands can be K-contiguous or M/N-contiguous.  Workgroups are
// renumbered so that the tiles resident on one XCD (the hardware deals
// workgroups to the 8 XCDs round-robin) form a contiguous block of the
// output, grouped 8 tiles down M, sharing A and B panels in that XCD's L2.
//
// bf16 path, other K (gemm_bf16_kernel): four waves of 128x128, tiles staged
// through registers with zero fill past M, N and K.
//
// fp32 path: a plain LDS-tiled FMA kernel (64x64 tile, 4x4 per thread), used
// by the fp32 workloads, whose matrices are small.
//
// Epilogues: plain fp32 store; bf16/fp32 store with a per-row bias; and the
// calibration-step forward epilogue (residual against the full-precision
// target, bf16 dL/dY, per-row partial sums of the squared residual and of dY).
#include <type_traits>

#include "common.h"
#include "oq_internal.h"

namespace oq {
namespace {

constexpr int BM = 256, BN = 256, BK = 64, NTHR = 256;
constexpr int GROUP_M = 8;
constexpr int F32_TILE = 64;

// ------------------------------------------------------------------ epilogues
// An epilogue sees the accumulators of one output row m in chunks of up to
// eight consecutive columns n .. n + cnt - 1: row(m) prepares the row,
// apply8 stores the chunk (16/32-byte vectors when vec) and returns its
// contributions to the row partials, finish writes one row's partials.
struct EpiF32 {
  float* C;
  int64_t ldc;
  bool vec;
  int64_t split_stride;              // elements between the K-split partial outputs
  static constexpr bool kRows = false;
  static constexpr bool kPre = false;
  OQ_DEV void split(int s) { C += s * split_stride; }
  struct Row { float* c; };
  OQ_DEV Row row(int64_t m) const { return Row{C + m * ldc}; }
  OQ_DEV float2 apply8(const Row& r, int64_t n, const float* v, int cnt) const {
    if (vec && cnt == 8) {
      store8(r.c + n, v);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (e < cnt) r.c[n + e] = v[e];
    }
    return make_float2(0.f, 0.f);
  }
  OQ_DEV void finish(int64_t, int, float, float) const {}
};

template <typename TC>
struct EpiStore {
  TC* C;
  int64_t ldc;
  const float* bias;
  bool vec;
  static constexpr bool kRows = false;
  static constexpr bool kPre = false;
  OQ_DEV void split(int) {}
  struct Row { TC* c; float b; };
  OQ_DEV Row row(int64_t m) const { return Row{C + m * ldc, bias ? bias[m] : 0.0f}; }
  OQ_DEV float2 apply8(const Row& r, int64_t n, const float* v, int cnt) const {
    float o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = v[e] + r.b;
    if (vec && cnt == 8) {
      store8(r.c + n, o);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (e < cnt) store1(r.c + n + e, o[e]);
    }
    return make_float2(0.f, 0.f);
  }
  OQ_DEV void finish(int64_t, int, float, float) const {}
};

// y = acc + B~[m]; r = y - y_fp; dY = r * 2/(T*c_out) stored in T;  row sums of r^2, dY.
// With a bf16 target the 8-wave kernel loads every chunk of y_fp a lane
// needs (pre) before it stages the accumulators, so the epilogue waits on
// one round of global loads instead of one per pass (apply8_pre).
template <typename T>
struct EpiResid {
  ResidArgs a;
  bool vec;
  static constexpr bool kRows = true;
  static constexpr bool kPre = sizeof(T) == 2;
  OQ_DEV void split(int) {}
  struct Row { const T* yfp; T* dy; float scale; float b; };
  OQ_DEV Row row(int64_t m) const {
    // constant indices only, so the argument block stays in scalar registers
    const void* y = a.yfp[0];
    float sc = a.scale[0];
    int64_t b = a.seg_begin[0];
#pragma unroll
    for (int s = 1; s < MAX_SEG; ++s) {
      if (s < a.nseg && m >= a.seg_begin[s]) {
        y = a.yfp[s];
        sc = a.scale[s];
        b = a.seg_begin[s];
      }
    }
    Row r;
    r.yfp = reinterpret_cast<const T*>(y) + (m - b) * a.ld_yfp;
    r.dy = reinterpret_cast<T*>(a.dy) + m * a.ld_dy;
    r.scale = sc;
    r.b = a.bias ? a.bias[m] : 0.0f;
    return r;
  }
  OQ_DEV float2 apply8(const Row& r, int64_t n, const float* v, int cnt) const {
    float yf[8];
    if (vec && cnt == 8) {
      load8(r.yfp + n, yf);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) yf[e] = e < cnt ? load1(r.yfp + n + e) : 0.0f;
    }
    return resid8(r, n, v, cnt, yf);
  }
  // bf16 target only: the raw chunk, then the chunk's arithmetic from it
  OQ_DEV uint4 pre(const Row& r, int64_t n, int cnt) const {
    if (vec && cnt == 8) return *reinterpret_cast<const uint4*>(r.yfp + n);
    uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (e < cnt) w[e >> 1] |= uint32_t(reinterpret_cast<const uint16_t*>(r.yfp)[n + e]) << (16 * (e & 1));
    return make_uint4(w[0], w[1], w[2], w[3]);
  }
  OQ_DEV float2 apply8_pre(const Row& r, int64_t n, const float* v, int cnt, uint4 q) const {
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
    float yf[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      yf[2 * e] = __uint_as_float(w[e] << 16);
      yf[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
    }
    return resid8(r, n, v, cnt, yf);
  }
  OQ_DEV float2 resid8(const Row& r, int64_t n, const float* v, int cnt, const float* yf) const {
    float d[8];
    const bool full = vec && cnt == 8;
    float sq = 0.f, sdy = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float y = v[e] + r.b;
      const float res = y - yf[e];
      d[e] = res * r.scale;
      if (e < cnt) {
        sq += res * res;
        sdy += rounded(d[e]);
      }
    }
    if (full) {
      store8(r.dy + n, d);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (e < cnt) store1(r.dy + n + e, d[e]);
    }
    return make_float2(sq, sdy);
  }
  OQ_DEV static float rounded(float d) {
    if constexpr (sizeof(T) == 2) return bf2f(f2bf(d));
    else return d;
  }
  OQ_DEV void finish(int64_t m, int tn, float sq, float dy) const {
    a.part_sq[m * a.ntn + tn] = sq;
    if (a.part_dy) a.part_dy[m * a.ntn + tn] = dy;
  }
};

// ------------------------------------------------------------------ bf16 epilogue
// The 128x128 fp32 quadrant of each wave goes through LDS in four passes of 32
// rows (row pitch 132 floats: the four row groups a fragment store touches
// land 16 banks apart), then every lane takes 8 consecutive columns of one
// row: global traffic is 16-byte vectors, 256 contiguous bytes per 16 lanes.
// Row partials: 8 columns per lane, a butterfly over the 16 lanes of the row,
// then the two waves of a tile row in a fixed order.
constexpr int EPI_PITCH = 132;

template <int P, class Epi>
OQ_DEV void epilogue_pass(f32x4_t (&acc)[8][8], const Epi& epi, int64_t m0, int64_t M, int wm,
                          int wn, int fr, int fk, int64_t nb, int cnt, float* reg,
                          float2 (*rowbuf)[BM]) {
#pragma unroll
  for (int ii = 0; ii < 2; ++ii)
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        reg[(16 * ii + 4 * fk + r) * EPI_PITCH + 16 * j + fr] = acc[2 * P + ii][j][r];
  for (int it = 0; it < 8; ++it) {
    const int rloc = fk + 4 * it;
    const int trow = wm * 128 + 32 * P + rloc;
    const int64_t m = m0 + trow;
    float v[8];
    const float4 a = *reinterpret_cast<const float4*>(reg + rloc * EPI_PITCH + 8 * fr);
    const float4 b = *reinterpret_cast<const float4*>(reg + rloc * EPI_PITCH + 8 * fr + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    float2 c = make_float2(0.f, 0.f);
    if (m < M && cnt > 0) c = epi.apply8(epi.row(m), nb, v, cnt);
    if constexpr (Epi::kRows) {
      c.x = group_sum<16>(c.x);
      c.y = group_sum<16>(c.y);
      if (fr == 0) rowbuf[wn][trow] = c;
    }
  }
}

template <class Epi>
OQ_DEV void epilogue_lds(f32x4_t (&acc)[8][8], const Epi& epi, int64_t m0, int64_t n0, int64_t M,
                         int64_t N, int tn, int wave, int lane, float* scratch,
                         float2 (*rowbuf)[BM]) {
  const int wm = wave >> 1, wn = wave & 1;
  const int fr = lane & 15, fk = lane >> 4;
  float* reg = scratch + wave * (32 * EPI_PITCH);
  const int64_t nb = n0 + wn * 128 + 8 * fr;
  const int cnt = int(max<int64_t>(0, min<int64_t>(8, N - nb)));
  epilogue_pass<0>(acc, epi, m0, M, wm, wn, fr, fk, nb, cnt, reg, rowbuf);
  epilogue_pass<1>(acc, epi, m0, M, wm, wn, fr, fk, nb, cnt, reg, rowbuf);
  epilogue_pass<2>(acc, epi, m0, M, wm, wn, fr, fk, nb, cnt, reg, rowbuf);
  epilogue_pass<3>(acc, epi, m0, M, wm, wn, fr, fk, nb, cnt, reg, rowbuf);
  if constexpr (Epi::kRows) {
    __syncthreads();
    const int tid = threadIdx.x;
    const int64_t m = m0 + tid;
    if (m < M) {
      float2 p0 = rowbuf[0][tid], p1 = rowbuf[1][tid];
      epi.finish(m, tn, p0.x + p1.x, p0.y + p1.y);
    }
  }
}

// ------------------------------------------------------------------ bf16 MFMA kernel
OQ_DEV bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

typedef __attribute__((address_space(1))) void gvoid_t;
typedef __attribute__((address_space(3))) void lvoid_t;

OQ_DEV void wait_vm0() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// 16-byte global -> LDS copy for every lane of the wave (lane i's bytes land
// at LDS byte address lds_addr + 16 i).  Issued as inline assembly so the
// compiler does not model it as an LDS write and adds no wait in front of
// the reads of the other stage; the kernel waits for it (vmcnt) itself
// before the barrier that publishes the stage.  m0 (the LDS base of the
// copy) is saved and restored around it, and one wait state separates the
// m0 write from the copy that reads it.
OQ_DEV void dma16(const void* g, uint32_t lds_addr) {
  const uint32_t m0v = __builtin_amdgcn_readfirstlane(lds_addr);
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
// The same copy with a uniform 64-bit base in SGPRs and a 32-bit per-lane
// byte offset (global address = base + offset).
OQ_DEV void dma16_s(const void* base, uint32_t vofs, uint32_t lds_addr) {
  const uint32_t m0v = __builtin_amdgcn_readfirstlane(lds_addr);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, %3\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(m0v), "v"(vofs), "s"(base)
      : "memory");
}
OQ_DEV uint32_t lds_addr_of(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>(
      (__attribute__((address_space(3))) const char*)(p)));
}

// DIRECT = true (K a multiple of 64): tiles go global -> LDS with
// global_load_lds_dwordx4, which writes lane i's 16 bytes at LDS base + 16 i.
// One such instruction fills 8 tile rows (64 slots); lane i fetches the global
// chunk that belongs in its slot, (i & 7) ^ row, so the LDS image is the same
// XOR-swizzled layout the fragment reads expect.  Rows past M (N) are clamped
// to the last valid row: they only feed output rows that are never stored.
// DIRECT = false: 16-byte loads through registers with zero fill past M, N, K.
template <class Epi, bool DIRECT>
__global__ __launch_bounds__(NTHR, 1) void gemm_bf16_kernel(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ B, int64_t M, int64_t N,
    int64_t K, int64_t lda, int64_t ldb, int tiles_m, int tiles_n, Epi epi) {
  __shared__ uint4 lds[2][2][BM * BK / 8];
  __shared__ float2 rowbuf[2][BM];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;

  // workgroup -> output tile: contiguous logical ranges per XCD, then
  // GROUP_M tile-rows swept column by column.
  const int nblk = gridDim.x, bid = blockIdx.x;
  const int xcd = bid & 7, local = bid >> 3, q = nblk >> 3, rem = nblk & 7;
  const int L = xcd * q + min(xcd, rem) + local;
  const int group_sz = GROUP_M * tiles_n;
  const int g = L / group_sz;
  const int first_m = g * GROUP_M;
  const int gm = min(GROUP_M, tiles_m - first_m);
  const int li = L - g * group_sz;
  const int tm = first_m + li % gm, tn = li / gm;
  const int64_t m0 = int64_t(tm) * BM, n0 = int64_t(tn) * BN;

  const int nk = int((K + BK - 1) / BK);

  // ---- per-thread load plan
  // DIRECT: instruction i of wave w fills tile rows 8 (4 i + w) .. +7; lane
  //   covers row 8 (4 i + w) + (lane >> 3), global chunk (lane & 7) ^ (lane >> 3).
  // register path: thread loads chunk (tid & 7) of rows (tid >> 3) + 32 i.
  int64_t aoff[8], boff[8];
  uint32_t amask = 0, bmask = 0;
  if constexpr (DIRECT) {
    const int r0 = 8 * wave + (lane >> 3);
    const int ch = (lane & 7) ^ (lane >> 3);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int64_t ra = min(m0 + r0 + 32 * i, M - 1);
      const int64_t rb = min(n0 + r0 + 32 * i, N - 1);
      aoff[i] = ra * lda + 8 * ch;
      boff[i] = rb * ldb + 8 * ch;
    }
  } else {
    const int lrow = tid >> 3, lch = tid & 7;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int64_t ra = m0 + lrow + 32 * i, rb = n0 + lrow + 32 * i;
      if (ra < M) amask |= 1u << i;
      if (rb < N) bmask |= 1u << i;
      aoff[i] = (ra < M ? ra : 0) * lda + 8 * lch;
      boff[i] = (rb < N ? rb : 0) * ldb + 8 * lch;
    }
  }
  const int sw_store = (tid & 7) ^ ((tid >> 3) & 7);   // register path slot

  const int wm = wave >> 1, wn = wave & 1;
  const int fr = lane & 15, fk = lane >> 4;

  f32x4_t acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  uint4 ra[8], rb[8];

  // ---- stage 0
  if constexpr (DIRECT) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      dma16(A + aoff[i], lds_addr_of(&lds[0][0][(4 * i + wave) * 64]));
      dma16(B + boff[i], lds_addr_of(&lds[0][1][(4 * i + wave) * 64]));
    }
    wait_vm0();
  } else {
    const bool kv = (tid & 7) * 8 < K;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      ra[i] = (kv && (amask >> i & 1u)) ? *reinterpret_cast<const uint4*>(A + aoff[i]) : make_uint4(0, 0, 0, 0);
      rb[i] = (kv && (bmask >> i & 1u)) ? *reinterpret_cast<const uint4*>(B + boff[i]) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      lds[0][0][((tid >> 3) + 32 * i) * 8 + sw_store] = ra[i];
      lds[0][1][((tid >> 3) + 32 * i) * 8 + sw_store] = rb[i];
    }
  }
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1, nxt = cur ^ 1;
    const bool more = kt + 1 < nk;
    const int64_t knext = int64_t(kt + 1) * BK;
    // 1. next stage in flight (the other LDS buffer, free since the last
    //    barrier): it has this whole iteration to arrive
    if (more) {
      if constexpr (DIRECT) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          dma16(A + aoff[i] + knext, lds_addr_of(&lds[nxt][0][(4 * i + wave) * 64]));
          dma16(B + boff[i] + knext, lds_addr_of(&lds[nxt][1][(4 * i + wave) * 64]));
        }
      } else {
        const bool kv = knext + (tid & 7) * 8 < K;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          ra[i] = (kv && (amask >> i & 1u)) ? *reinterpret_cast<const uint4*>(A + aoff[i] + knext)
                                            : make_uint4(0, 0, 0, 0);
          rb[i] = (kv && (bmask >> i & 1u)) ? *reinterpret_cast<const uint4*>(B + boff[i] + knext)
                                            : make_uint4(0, 0, 0, 0);
        }
      }
    }
    // 2. the whole K-slice of this wave's fragments into registers
    const uint4* As = lds[cur][0];
    const uint4* Bs = lds[cur][1];
    bf16x8_t af[2][8], bfr[2][8];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int ch = (kk * 4 + fk) ^ (fr & 7);
#pragma unroll
      for (int i = 0; i < 8; ++i) af[kk][i] = as_bf16x8(As[(wm * 128 + 16 * i + fr) * 8 + ch]);
#pragma unroll
      for (int j = 0; j < 8; ++j) bfr[kk][j] = as_bf16x8(Bs[(wn * 128 + 16 * j + fr) * 8 + ch]);
    }
    // 3. 128 matrix instructions on the registers
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[kk][i], bfr[kk][j], acc[i][j], 0, 0, 0);
    // 4. next stage complete and visible to every wave
    if (more) {
      if constexpr (DIRECT) {
        wait_vm0();
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          lds[nxt][0][((tid >> 3) + 32 * i) * 8 + sw_store] = ra[i];
          lds[nxt][1][((tid >> 3) + 32 * i) * 8 + sw_store] = rb[i];
        }
      }
    }
    __syncthreads();
  }

  // the loop ended with a barrier: every LDS read is done
  epilogue_lds(acc, epi, m0, n0, M, N, tn, wave, lane, reinterpret_cast<float*>(&lds[0][0][0]),
               rowbuf);
}

// ------------------------------------------------------------------ bf16 8-wave kernel
// K % 64 == 0.  The same 256x256x64 tile as above, but eight waves (two per
// SIMD) each own a 128x64 block (2 x 4 waves): while one wave of a SIMD waits
// the other issues matrix instructions.
// K-major LDS slot of chunk c of row r: c ^ (r & 7) ^ ((r >> 4) & 1).  A
// 128-bit LDS read serves lanes 0-7 together with 16-23 (and so on); the
// row-bit-4 term keeps rows r and r + 16 apart as well.
constexpr int NTHR8 = 512;
constexpr int EPI8_PITCH = 68;

// Operand tiles.  An operand is K-major (rows of the M or N side, k
// contiguous: the A and B of C = A B^T) or MN-major (rows of k, the M or N
// side contiguous).  Either way a stage's tile is 32 KiB:
//  * K-major: 256 rows x 64 k, eight 16-byte chunks per row, chunk c of row r
//    at slot c ^ (r & 7) ^ ((r >> 4) & 1);
//  * MN-major: 64 k-rows x 256, 32 chunks per row, chunk c of k-row r at slot
//    c ^ 2 h(r) with h(r) = (r & 3) | ((r >> 3) & 1) << 2.  A fragment takes
//    two ds_read_b64_tr_b16 (4 k each); the swizzle puts the eight k-rows one
//    such read touches in eight different 32-byte bank groups.
// ds_read_b64_tr_b16: within each 16-lane group, with M[j] the four 16-bit
// values at lane j's address, lane i receives M[4 e + i / 4][i % 4], e = 0..3.
// Lane j = 4 e + i / 4 therefore points at k-row k0 + j / 4, column
// 16 q + 4 (j % 4), and lane i receives k0 .. k0 + 3 of column 16 q + i.
OQ_DEV int mn_swz(int r) { return (r & 3) | (((r >> 3) & 1) << 2); }

// Per-lane byte offsets of a stage's four DMA instructions for one operand,
// from the operand's tile origin (row mn0 for K-major, column mn0 for
// MN-major).  Rows (K-major) or columns (MN-major) past the operand's extent
// are clamped to the last valid one: they feed only outputs never stored.
template <bool MN>
OQ_DEV void dma_plan(uint32_t (&off)[4], int64_t mn0, int64_t extent, int64_t ld, int wave,
                     int lane) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if constexpr (MN) {
      // instruction i of wave w fills k-rows 2 (8 i + w) and +1 (512 bytes each)
      const int r = 16 * i + 2 * wave + (lane >> 5);
      const int c = (lane & 31) ^ (2 * mn_swz(r));
      const int64_t col = min<int64_t>(8 * c, extent - 8 - mn0);
      off[i] = uint32_t(2 * (r * ld + col));
    } else {
      // instruction i of wave w fills rows 8 (8 i + w) .. +7 (128 bytes each)
      const int row = 64 * i + 8 * wave + (lane >> 3);
      const int c = (lane & 7) ^ (lane >> 3) ^ ((wave >> 1) & 1);
      off[i] = uint32_t(2 * (min<int64_t>(row, extent - 1 - mn0) * ld + 8 * c));
    }
  }
}

typedef const __attribute__((address_space(3))) char lds_cchar;

// One fragment (16 rows of the M/N side x 32 k, k-half kk) of the tile at
// tile; q = first row / 16.
template <bool MN>
OQ_DEV bf16x8_t frag(lds_cchar* tile, int q, int kk, int lane) {
  typedef short v4i16 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) v4i16 lds_v4;
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  typedef const __attribute__((address_space(3))) u32x4 lds_u4;
  if constexpr (MN) {
    const int g = lane >> 4, j = lane & 15;
    lds_cchar* a = tile + kk * 16384 + g * 4096 + (j >> 2) * 512 + 8 * (j & 3) +
                   32 * (q ^ mn_swz(8 * g + (j >> 2)));
    const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4*)a);
    const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4*)(a + 2048));
    return __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  } else {
    const int row = 16 * q + (lane & 15);
    const int slot = (kk * 4 + (lane >> 4)) ^ (row & 7) ^ ((row >> 4) & 1);
    return __builtin_bit_cast(bf16x8_t, reinterpret_cast<lds_u4*>(tile)[row * 8 + slot]);
  }
}

OQ_DEV void mfma_half(f32x4_t (&acc)[8][4], const bf16x8_t (&af)[8], const bf16x8_t (&bq)[4]) {
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bq[j], acc[i][j], 0, 0, 0);
}

// Epilogue of the 8-wave kernels: each wave's 128x64 block goes through LDS
// (scratch, 8 x 32 x EPI8_PITCH floats) in four passes of 32 rows; a lane
// then takes 8 consecutive columns of one row (8 lanes per row).  Row
// partials: 8 lanes per row, then the four column waves in a fixed order.
template <int P, class Epi>
OQ_DEV void epi8_pass(const f32x4_t (&acc)[8][4], const Epi& epi, int64_t m0, int64_t M, int wm,
                      int wn, int lane, int64_t nb, int cnt, float* reg, float2 (*rowbuf)[BM],
                      const uint4 (&pre)[4][4]) {
  constexpr int PITCH = EPI8_PITCH;
  const int fr = lane & 15, fk = lane >> 4;
  const int cl = lane & 7, rl = lane >> 3;
#pragma unroll
  for (int ii = 0; ii < 2; ++ii)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        reg[(16 * ii + 4 * fk + r) * PITCH + 16 * j + fr] = acc[2 * P + ii][j][r];
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const int rloc = rl + 8 * it;
    const int trow = wm * 128 + 32 * P + rloc;
    const int64_t m = m0 + trow;
    float v[8];
    const float4 a_ = *reinterpret_cast<const float4*>(reg + rloc * PITCH + 8 * cl);
    const float4 b_ = *reinterpret_cast<const float4*>(reg + rloc * PITCH + 8 * cl + 4);
    v[0] = a_.x; v[1] = a_.y; v[2] = a_.z; v[3] = a_.w;
    v[4] = b_.x; v[5] = b_.y; v[6] = b_.z; v[7] = b_.w;
    float2 c = make_float2(0.f, 0.f);
    if (m < M && cnt > 0) {
      if constexpr (Epi::kPre) c = epi.apply8_pre(epi.row(m), nb, v, cnt, pre[P][it]);
      else c = epi.apply8(epi.row(m), nb, v, cnt);
    }
    if constexpr (Epi::kRows) {
      c.x = group_sum<8>(c.x);
      c.y = group_sum<8>(c.y);
      if (cl == 0) rowbuf[wn][trow] = c;
    }
  }
}

// fp32 store epilogue, fast form (a tile inside N, 16-byte access): a lane
// stores columns 4 c .. 4 c + 3 and 32 + 4 c .. 32 + 4 c + 3 of its row, so
// each store instruction writes 128 contiguous bytes per row (the general
// form's 8 consecutive columns per lane make every instruction cover half of
// each 32-byte piece).
OQ_DEV void epilogue8_f32(const f32x4_t (&acc)[8][4], const EpiF32& epi, int64_t m0, int64_t n0,
                          int64_t M, int wave, int lane, float* scratch) {
  constexpr int PITCH = EPI8_PITCH;
  const int wm = wave >> 2, wn = wave & 3;
  float* reg = scratch + wave * (32 * PITCH);
  const int fr = lane & 15, fk = lane >> 4;
  const int cl = lane & 7, rl = lane >> 3;
  float* cb = epi.C + (m0 + wm * 128 + rl) * epi.ldc + n0 + wn * 64 + 4 * cl;
#pragma unroll
  for (int P = 0; P < 4; ++P) {
#pragma unroll
    for (int ii = 0; ii < 2; ++ii)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          reg[(16 * ii + 4 * fk + r) * PITCH + 16 * j + fr] = acc[2 * P + ii][j][r];
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int rloc = rl + 8 * it;
      if (m0 + wm * 128 + 32 * P + rloc < M) {
        const float4 lo = *reinterpret_cast<const float4*>(reg + rloc * PITCH + 4 * cl);
        const float4 hi = *reinterpret_cast<const float4*>(reg + rloc * PITCH + 32 + 4 * cl);
        float* c = cb + int64_t(32 * P + 8 * it) * epi.ldc;
        *reinterpret_cast<float4*>(c) = lo;
        *reinterpret_cast<float4*>(c + 32) = hi;
      }
    }
  }
}

template <class Epi>
OQ_DEV void epilogue8(const f32x4_t (&acc)[8][4], const Epi& epi, int64_t m0, int64_t n0,
                      int64_t M, int64_t N, int tn, int wave, int lane, float* scratch,
                      float2 (*rowbuf)[BM]) {
  const int wm = wave >> 2, wn = wave & 3;
  float* reg = scratch + wave * (32 * EPI8_PITCH);
  const int64_t nb = n0 + wn * 64 + 8 * (lane & 7);
  const int cnt = int(max<int64_t>(0, min<int64_t>(8, N - nb)));
  // the chunks of every pass in flight at once (row m0 + wm 128 + 32 P + lane/8 + 8 it)
  uint4 pre[4][4];
  if constexpr (Epi::kPre) {
#pragma unroll
    for (int P = 0; P < 4; ++P)
#pragma unroll
      for (int it = 0; it < 4; ++it) {
        const int64_t m = m0 + wm * 128 + 32 * P + (lane >> 3) + 8 * it;
        pre[P][it] = (m < M && cnt > 0) ? epi.pre(epi.row(m), nb, cnt) : make_uint4(0u, 0u, 0u, 0u);
      }
  }
  epi8_pass<0>(acc, epi, m0, M, wm, wn, lane, nb, cnt, reg, rowbuf, pre);
  epi8_pass<1>(acc, epi, m0, M, wm, wn, lane, nb, cnt, reg, rowbuf, pre);
  epi8_pass<2>(acc, epi, m0, M, wm, wn, lane, nb, cnt, reg, rowbuf, pre);
  epi8_pass<3>(acc, epi, m0, M, wm, wn, lane, nb, cnt, reg, rowbuf, pre);
  if constexpr (Epi::kRows) {
    __syncthreads();
    const int tid = threadIdx.x;
    if (tid < BM) {
      const int64_t m = m0 + tid;
      if (m < M) {
        float2 s = rowbuf[0][tid];
#pragma unroll
        for (int w = 1; w < 4; ++w) {
          s.x += rowbuf[w][tid].x;
          s.y += rowbuf[w][tid].y;
        }
        epi.finish(m, tn, s.x, s.y);
      }
    }
  }
}

// Residual epilogue, fast form, for a tile inside M and N whose rows all
// belong to one stacked linear, with 16-byte access: the linear is looked up
// once per tile, a lane's 16 rows are its first row plus constant strides,
// their bias and target chunks are loaded before the accumulators are
// staged, and the 8-lane row sums run on DPP (quad xor 1, quad xor 2, then
// the half-row mirror: the same pairings as the butterfly, so the sums are
// bit-identical to the general form's).
template <int L>
OQ_DEV float group_sum_dpp(float v) {
  static_assert(L == 1 || L == 2 || L == 4 || L == 8, "groups of up to 8 lanes");
  if constexpr (L >= 2) v += dpp_f(v, 0);
  if constexpr (L >= 4) v += dpp_f(v, 1);
  if constexpr (L >= 8) v += dpp_f(v, 2);
  return v;
}
OQ_DEV float group8_sum(float v) { return group_sum_dpp<8>(v); }

OQ_DEV int resid_seg(const ResidArgs& a, int64_t m) {
  int s = 0;
#pragma unroll
  for (int k = 1; k < MAX_SEG; ++k)
    if (k < a.nseg && m >= a.seg_begin[k]) s = k;
  return s;
}

// BIAS: the tile's linear has a bias; DY: the row sums of dY are wanted
// (the LET bias path).  Without them their per-element work is not done.
template <bool BIAS, bool DY>
OQ_DEV void epilogue8_resid(const f32x4_t (&acc)[8][4], const EpiResid<uint16_t>& ep, int seg,
                            int64_t m0, int64_t n0, int tn, int wave, int lane, float* scratch,
                            float2 (*rowbuf)[BM]) {
  constexpr int PITCH = EPI8_PITCH;
  const ResidArgs& a = ep.a;
  const int wm = wave >> 2, wn = wave & 3;
  const int fr = lane & 15, fk = lane >> 4;
  const int cl = lane & 7, rl = lane >> 3;
  float* reg = scratch + wave * (32 * PITCH);
  // this lane's first row m0 + wm 128 + rl; the others follow at 32 P + 8 it
  const int64_t mr = m0 + wm * 128 + rl;
  const int64_t nb = n0 + wn * 64 + 8 * cl;
  const float scale = a.scale[seg];
  const uint16_t* yl = static_cast<const uint16_t*>(a.yfp[seg]) + (mr - a.seg_begin[seg]) * a.ld_yfp + nb;
  uint16_t* dl = static_cast<uint16_t*>(a.dy) + mr * a.ld_dy + nb;
  uint4 yv[4][4];
  float bv[4][4];
#pragma unroll
  for (int P = 0; P < 4; ++P)
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int64_t o = 32 * P + 8 * it;
      yv[P][it] = *reinterpret_cast<const uint4*>(yl + o * a.ld_yfp);
      bv[P][it] = BIAS ? a.bias[mr + o] : 0.0f;
    }
#pragma unroll
  for (int P = 0; P < 4; ++P) {
#pragma unroll
    for (int ii = 0; ii < 2; ++ii)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          reg[(16 * ii + 4 * fk + r) * PITCH + 16 * j + fr] = acc[2 * P + ii][j][r];
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int rloc = rl + 8 * it;
      const float4 lo = *reinterpret_cast<const float4*>(reg + rloc * PITCH + 8 * cl);
      const float4 hi = *reinterpret_cast<const float4*>(reg + rloc * PITCH + 8 * cl + 4);
      const float v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
      const uint32_t w[4] = {yv[P][it].x, yv[P][it].y, yv[P][it].z, yv[P][it].w};
      float d[8], sq = 0.f, sdy = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float yf = __uint_as_float(e & 1 ? w[e >> 1] & 0xffff0000u : w[e >> 1] << 16);
        const float res = (BIAS ? v[e] + bv[P][it] : v[e]) - yf;
        d[e] = res * scale;
        sq += res * res;
        if (DY) sdy += bf2f(f2bf(d[e]));
      }
      store8(dl + int64_t(32 * P + 8 * it) * a.ld_dy, d);
      sq = group8_sum(sq);
      if (DY) sdy = group8_sum(sdy);
      if (cl == 0) rowbuf[wn][wm * 128 + 32 * P + rloc] = make_float2(sq, sdy);
    }
  }
  __syncthreads();
  const int tid = threadIdx.x;
  if (tid < BM) {
    float2 t = rowbuf[0][tid];
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      t.x += rowbuf[w][tid].x;
      t.y += rowbuf[w][tid].y;
    }
    ep.finish(m0 + tid, tn, t.x, t.y);
  }
}

// Weight gradient with the LWC straight-through backward fused (no LET):
// the accumulators are dW^ for rows m (output channels of the stacked
// linears) and columns n (input channels).  G = group / 8 lanes of a row
// cover one group; groups of 128 and 256 span two and four column waves and
// meet in LDS.
template <int G>
struct EpiLwc {
  LwcArgs a;
  static constexpr bool kRows = false;
  OQ_DEV void split(int) {}
  // linear of stacked row m: constant indices only, so the argument block
  // stays in scalar registers
  // (o: m's row within its linear, b: the linear's first stacked row)
  struct Seg { const uint16_t* w; float* dgl; float* dbl; int64_t o, b; };
  OQ_DEV Seg seg(int64_t m) const {
    Seg s{a.W[0], a.dgl[0], a.dbl[0], m - a.seg_begin[0], a.seg_begin[0]};
#pragma unroll
    for (int i = 1; i < MAX_SEG; ++i) {
      if (i < a.nseg && m >= a.seg_begin[i]) {
        s = Seg{a.W[i], a.dgl[i], a.dbl[i], m - a.seg_begin[i], a.seg_begin[i]};
      }
    }
    return s;
  }
  // S_h, S_z of one 8-column chunk of row m at column n
  OQ_DEV float2 chunk(int64_t m, int64_t n, const float* g) const {
    const Seg s = seg(m);
    float w[8];
    load8(s.w + s.o * a.C + n, w);
    const int64_t gi = m * a.ng + n / a.group;
    return chunk_terms(w, g, a.gstat[2 * gi].w, a.gstat[2 * gi + 1].z);
  }
  // the same from the chunk's weights, the group's z and 1/h
  OQ_DEV float2 chunk_terms(const float* w, const float* g, float z, float r) const {
    const float lo = -z, hi = a.qmax - z;
    float2 c = make_float2(0.f, 0.f);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      // q - z = med3(rint(u), -z, qmax - z); inside the clamp exactly when
      // the median left rint(u) alone
      const float u = w[e] * r;
      const float ru = rintf(u);
      const float tq = __builtin_amdgcn_fmed3f(ru, lo, hi);
      const bool in = tq == ru;
      c.x += g[e] * (in ? tq - u : tq);
      c.y += in ? 0.0f : g[e];
    }
    return c;
  }
  // Eq. 2's parameters again from the group's max / min and the clip
  // strengths the forward recorded, then the logit gradients
  OQ_DEV void finish(int64_t m, int gi, float sh, float sz) const { finish_in(seg(m), m, gi, sh, sz); }
  OQ_DEV void finish_in(const Seg& s, int64_t m, int gi, float sh, float sz) const {
    const float4 st = a.gstat[2 * (m * a.ng + gi)];
    const float4 gb = a.gstat[2 * (m * a.ng + gi) + 1];
    const int64_t k = (m - s.b) * a.ng + gi;
    const QParams p = make_qparams(st.x, st.y, gb.x, gb.y, a.qmax);
    const QGrad qg = quant_group_grad(sh, sz, st.x, st.y, p, a.qmax);
    s.dgl[k] = qg.dgamma * p.gamma * (1.0f - p.gamma);
    s.dbl[k] = qg.dbeta * p.beta * (1.0f - p.beta);
  }
};

template <class E>
struct IsLwc : std::false_type {};
template <int G>
struct IsLwc<EpiLwc<G>> : std::true_type {};

template <int G>
OQ_DEV void epilogue8_lwc(const f32x4_t (&acc)[8][4], const EpiLwc<G>& ep, int64_t m0,
                          int64_t n0, int64_t M, int64_t N, int wave, int lane, float* scratch,
                          float2 (*rowbuf)[BM]) {
  constexpr int PITCH = EPI8_PITCH;
  const int wm = wave >> 2, wn = wave & 3;
  float* reg = scratch + wave * (32 * EPI8_PITCH);
  const int fr = lane & 15, fk = lane >> 4;
  const int cl = lane & 7, rl = lane >> 3;
  const int64_t nb = n0 + wn * 64 + 8 * cl;
  const bool colok = nb < N;                 // N % 8 == 0: a chunk is whole or absent
#pragma unroll
  for (int P = 0; P < 4; ++P) {
#pragma unroll
    for (int ii = 0; ii < 2; ++ii)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          reg[(16 * ii + 4 * fk + r) * PITCH + 16 * j + fr] = acc[2 * P + ii][j][r];
    for (int it = 0; it < 4; ++it) {
      const int rloc = rl + 8 * it;
      const int trow = wm * 128 + 32 * P + rloc;
      const int64_t m = m0 + trow;
      float2 c = make_float2(0.f, 0.f);
      if (m < M && colok) {
        float v[8];
        const float4 a_ = *reinterpret_cast<const float4*>(reg + rloc * PITCH + 8 * cl);
        const float4 b_ = *reinterpret_cast<const float4*>(reg + rloc * PITCH + 8 * cl + 4);
        v[0] = a_.x; v[1] = a_.y; v[2] = a_.z; v[3] = a_.w;
        v[4] = b_.x; v[5] = b_.y; v[6] = b_.z; v[7] = b_.w;
        c = ep.chunk(m, nb, v);
      }
      if constexpr (G <= 8) {
        c.x = group_sum<G>(c.x);
        c.y = group_sum<G>(c.y);
        if (m < M && colok && cl % G == 0) ep.finish(m, int(nb / ep.a.group), c.x, c.y);
      } else {
        c.x = group_sum<8>(c.x);
        c.y = group_sum<8>(c.y);
        if (cl == 0) rowbuf[wn][trow] = c;
      }
    }
  }
  if constexpr (G > 8) {
    // a group covers WPG column waves; GPR groups per tile row
    constexpr int WPG = G / 8, GPR = 4 / WPG;
    __syncthreads();
    for (int idx = threadIdx.x; idx < BM * GPR; idx += NTHR8) {
      const int trow = idx / GPR, gq = idx % GPR;
      const int64_t m = m0 + trow, ng0 = n0 + int64_t(gq) * WPG * 64;
      if (m < M && ng0 < N) {
        float2 s = rowbuf[gq * WPG][trow];
#pragma unroll
        for (int w = 1; w < WPG; ++w) {
          s.x += rowbuf[gq * WPG + w][trow].x;
          s.y += rowbuf[gq * WPG + w][trow].y;
        }
        ep.finish(m, int(ng0 / ep.a.group), s.x, s.y);
      }
    }
  }
}

// Fused LWC epilogue, fast form, for a tile inside M and N whose rows all
// belong to one linear: the linear is looked up once, and every weight chunk
// and group record a lane needs (its 16 rows at constant strides) is loaded
// before the accumulators are staged, so the epilogue waits on one round of
// loads instead of one per pass.
template <int G>
OQ_DEV void epilogue8_lwc_fast(const f32x4_t (&acc)[8][4], const EpiLwc<G>& ep,
                               const typename EpiLwc<G>::Seg& sg, int64_t m0, int64_t n0, int wave,
                               int lane, float* scratch, float2 (*rowbuf)[BM]) {
  constexpr int PITCH = EPI8_PITCH;
  const LwcArgs& a = ep.a;
  const int wm = wave >> 2, wn = wave & 3;
  float* reg = scratch + wave * (32 * EPI8_PITCH);
  const int fr = lane & 15, fk = lane >> 4;
  const int cl = lane & 7, rl = lane >> 3;
  const int64_t mr = m0 + wm * 128 + rl;     // this lane's first row; the others at 32 P + 8 it
  const int64_t nb = n0 + wn * 64 + 8 * cl;
  const int gi = int(nb / a.group);
  const uint16_t* wl = sg.w + (mr - sg.b) * a.C + nb;
  const float* rec = reinterpret_cast<const float*>(a.gstat) + 8 * (mr * a.ng + gi);
  uint4 wv[4][4];
  float zv[4][4], rv[4][4];
#pragma unroll
  for (int P = 0; P < 4; ++P)
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int64_t o = 32 * P + 8 * it;
      wv[P][it] = *reinterpret_cast<const uint4*>(wl + o * a.C);
      zv[P][it] = rec[8 * o * a.ng + 3];
      rv[P][it] = rec[8 * o * a.ng + 6];
    }
#pragma unroll
  for (int P = 0; P < 4; ++P) {
#pragma unroll
    for (int ii = 0; ii < 2; ++ii)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          reg[(16 * ii + 4 * fk + r) * PITCH + 16 * j + fr] = acc[2 * P + ii][j][r];
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int rloc = rl + 8 * it;
      const int trow = wm * 128 + 32 * P + rloc;
      const float4 lo = *reinterpret_cast<const float4*>(reg + rloc * PITCH + 8 * cl);
      const float4 hi = *reinterpret_cast<const float4*>(reg + rloc * PITCH + 8 * cl + 4);
      const float g[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
      const uint32_t ww[4] = {wv[P][it].x, wv[P][it].y, wv[P][it].z, wv[P][it].w};
      float w[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        w[2 * e] = __uint_as_float(ww[e] << 16);
        w[2 * e + 1] = __uint_as_float(ww[e] & 0xffff0000u);
      }
      float2 c = ep.chunk_terms(w, g, zv[P][it], rv[P][it]);
      // DPP sums with the butterfly's pairings (bit-identical)
      if constexpr (G <= 8) {
        c.x = group_sum_dpp<G>(c.x);
        c.y = group_sum_dpp<G>(c.y);
        if (cl % G == 0) ep.finish_in(sg, m0 + trow, gi, c.x, c.y);
      } else {
        c.x = group_sum_dpp<8>(c.x);
        c.y = group_sum_dpp<8>(c.y);
        if (cl == 0) rowbuf[wn][trow] = c;
      }
    }
  }
  if constexpr (G > 8) {
    constexpr int WPG = G / 8, GPR = 4 / WPG;
    __syncthreads();
    for (int idx = threadIdx.x; idx < BM * GPR; idx += NTHR8) {
      const int trow = idx / GPR, gq = idx % GPR;
      float2 t = rowbuf[gq * WPG][trow];
#pragma unroll
      for (int w = 1; w < WPG; ++w) {
        t.x += rowbuf[gq * WPG + w][trow].x;
        t.y += rowbuf[gq * WPG + w][trow].y;
      }
      ep.finish_in(sg, m0 + trow, int((n0 + int64_t(gq) * WPG * 64) / a.group), t.x, t.y);
    }
  }
}

// Stages: B's tile of stage s in one of three buffers (s % 3), A's in one of
// two (s % 2), 160 KiB in all.  Iteration kt runs k-half 1 of stage kt, then
// (after the middle barrier) k-half 0 of stage kt + 1.  B's buffer for stage
// kt + 2 held stage kt - 1 and is free during the whole iteration, so its
// copies go into the first k-half; A's held stage kt and is free after the
// middle barrier, so its copies go into the second.  Each half then carries
// 32 KiB of copies rather than one half carrying 64 (the per-CU copy path
// moves about 64 bytes a clock), and B's copies have one and a half
// iterations to land.
template <bool AMN, bool BMN>
OQ_DEV void read_frags(lds_cchar* at, lds_cchar* bt, int kk, int wm, int wn, int lane,
                       bf16x8_t (&af)[8], bf16x8_t (&bq)[4]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) af[i] = frag<AMN>(at, 8 * wm + i, kk, lane);
#pragma unroll
  for (int j = 0; j < 4; ++j) bq[j] = frag<BMN>(bt, 4 * wn + j, kk, lane);
}

// One k-half: 8 groups of four MFMAs; the next fragment set's 12 reads in
// groups 0..5 (B first), and when DMA one copy of an operand tile (base Xb,
// offsets xoff, LDS tile at wr) in each even group.
template <bool AMN, bool BMN, bool DMA>
OQ_DEV void half_sched(f32x4_t (&acc)[8][4], const bf16x8_t (&au)[8], const bf16x8_t (&bu)[4],
                       lds_cchar* ra, lds_cchar* rb, int kk, int wm, int wn, int lane,
                       bf16x8_t (&ad)[8], bf16x8_t (&bd)[4], const uint16_t* Xb,
                       const uint32_t (&xoff)[4], uint32_t wr, int wave) {
#pragma unroll
  for (int g = 0; g < 8; ++g) {
    if (g < 2) {
      bd[2 * g] = frag<BMN>(rb, 4 * wn + 2 * g, kk, lane);
      bd[2 * g + 1] = frag<BMN>(rb, 4 * wn + 2 * g + 1, kk, lane);
    } else if (g < 6) {
      ad[2 * g - 4] = frag<AMN>(ra, 8 * wm + 2 * g - 4, kk, lane);
      ad[2 * g - 3] = frag<AMN>(ra, 8 * wm + 2 * g - 3, kk, lane);
    }
    if constexpr (DMA) {
      if ((g & 1) == 0) dma16_s(Xb, xoff[g >> 1], wr + (8 * (g >> 1) + wave) * 1024);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
      acc[g][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(au[g], bu[j], acc[g][j], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
}

OQ_DEV void wait_vm4() { asm volatile("s_waitcnt vmcnt(4)" ::: "memory"); }

template <class Epi, bool AMN, bool BMN>
__global__ __launch_bounds__(NTHR8, 1) void gemm_bf16_w8_kernel(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ B, int64_t M, int64_t N,
    int64_t K, int64_t lda, int64_t ldb, int tiles_m, int tiles_n, Epi epi) {
  // With a K split (grid = tiles x splits) each workgroup runs K of the
  // whole and writes its own partial output (Epi::split).
  // B stages at 0, 32 and 64 KiB, A stages at 96 and 128 KiB
  __shared__ uint4 lds[5 * 32768 / 16];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int nblk = gridDim.x, bid = blockIdx.x;
  const int xcd = bid & 7, local = bid >> 3, q = nblk >> 3, rem = nblk & 7;
  const int Lall = xcd * q + min(xcd, rem) + local;
  const int ks = Lall / (tiles_m * tiles_n);
  const int L = Lall - ks * (tiles_m * tiles_n);
  const int group_sz = GROUP_M * tiles_n;
  const int g = L / group_sz;
  const int first_m = g * GROUP_M;
  const int gm = min(GROUP_M, tiles_m - first_m);
  const int li = L - g * group_sz;
  const int tm = first_m + li % gm, tn = li / gm;
  const int64_t m0 = int64_t(tm) * BM, n0 = int64_t(tn) * BN;
  const int nk = int(K / BK);
  if (ks) {
    A += AMN ? ks * K * lda : ks * K;
    B += BMN ? ks * K * ldb : ks * K;
    epi.split(ks);
  }

  const uint16_t* At = AMN ? A + m0 : A + m0 * lda;
  const uint16_t* Bt = BMN ? B + n0 : B + n0 * ldb;
  const int64_t astep = AMN ? BK * lda : BK, bstep = BMN ? BK * ldb : BK;
  uint32_t aoff[4], boff[4];
  dma_plan<AMN>(aoff, m0, M, lda, wave, lane);
  dma_plan<BMN>(boff, n0, N, ldb, wave, lane);
  const uint32_t lds0 = lds_addr_of(&lds[0]);
  lds_cchar* lbase = (lds_cchar*)(&lds[0]);
  const int wm = wave >> 2, wn = wave & 3;
  auto b_lds = [&](int s) { return lds0 + uint32_t(s % 3) * 32768u; };
  auto a_lds = [&](int s) { return lds0 + 98304u + uint32_t(s & 1) * 32768u; };
  auto b_tile = [&](int s) { return lbase + (s % 3) * 32768; };
  auto a_tile = [&](int s) { return lbase + 98304 + (s & 1) * 32768; };

  f32x4_t acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) acc[i][j][v] = 0.f;

  // stage 0 (A then B), then stage 1 in flight
#pragma unroll
  for (int i = 0; i < 4; ++i) dma16_s(At, aoff[i], a_lds(0) + (8 * i + wave) * 1024);
#pragma unroll
  for (int i = 0; i < 4; ++i) dma16_s(Bt, boff[i], b_lds(0) + (8 * i + wave) * 1024);
  wait_vm0();
  __syncthreads();
  bf16x8_t a0[8], b0[4], a1[8], b1[4];
  read_frags<AMN, BMN>(a_tile(0), b_tile(0), 0, wm, wn, lane, a0, b0);
  if (nk > 1) {
#pragma unroll
    for (int i = 0; i < 4; ++i) dma16_s(At + astep, aoff[i], a_lds(1) + (8 * i + wave) * 1024);
#pragma unroll
    for (int i = 0; i < 4; ++i) dma16_s(Bt + bstep, boff[i], b_lds(1) + (8 * i + wave) * 1024);
  }

  // iteration kt: the first half copies B of stage kt + 2 (its buffer held
  // stage kt - 1), the second half A of stage kt + 2 (its buffer held stage
  // kt, whose last reads end at the middle barrier); the middle barrier
  // waits for stage kt + 1 with B of stage kt + 2 still in flight.
  int kt = 0;
  for (; kt + 2 < nk; ++kt) {
    half_sched<AMN, BMN, true>(acc, a0, b0, a_tile(kt), b_tile(kt), 1, wm, wn, lane, a1, b1,
                               Bt + (kt + 2) * bstep, boff, b_lds(kt + 2), wave);
    wait_vm4();
    __syncthreads();
    half_sched<AMN, BMN, true>(acc, a1, b1, a_tile(kt + 1), b_tile(kt + 1), 0, wm, wn, lane, a0,
                               b0, At + (kt + 2) * astep, aoff, a_lds(kt + 2), wave);
  }
  for (; kt < nk; ++kt) {
    read_frags<AMN, BMN>(a_tile(kt), b_tile(kt), 1, wm, wn, lane, a1, b1);
    mfma_half(acc, a0, b0);
    if (kt + 1 < nk) wait_vm0();
    __syncthreads();
    if (kt + 1 < nk) read_frags<AMN, BMN>(a_tile(kt + 1), b_tile(kt + 1), 0, wm, wn, lane, a0, b0);
    mfma_half(acc, a1, b1);
  }
  __syncthreads();
  // epilogue staging (68 KiB) and row partials (8 KiB at 96 KiB) reuse the stages
  if constexpr (IsLwc<Epi>::value) {
    float* stg = reinterpret_cast<float*>(&lds[0]);
    auto rows = reinterpret_cast<float2 (*)[BM]>(reinterpret_cast<char*>(&lds[0]) + 98304);
    // the fast form when the tile is whole and within one linear (uniform)
    const auto sg = epi.seg(m0);
    if (m0 + BM <= M && n0 + BN <= N && epi.seg(m0 + BM - 1).b == sg.b)
      epilogue8_lwc_fast(acc, epi, sg, m0, n0, wave, lane, stg, rows);
    else
      epilogue8_lwc(acc, epi, m0, n0, M, N, wave, lane, stg, rows);
  } else {
    float* stg = reinterpret_cast<float*>(&lds[0]);
    auto rows = reinterpret_cast<float2 (*)[BM]>(reinterpret_cast<char*>(&lds[0]) + 98304);
    if constexpr (std::is_same<Epi, EpiResid<uint16_t>>::value) {
      // the fast form when the tile is whole and within one linear (uniform)
      const int seg = resid_seg(epi.a, m0);
      if (epi.vec && m0 + BM <= M && n0 + BN <= N && resid_seg(epi.a, m0 + BM - 1) == seg) {
        if (epi.a.bias) {
          if (epi.a.part_dy) epilogue8_resid<true, true>(acc, epi, seg, m0, n0, tn, wave, lane, stg, rows);
          else epilogue8_resid<true, false>(acc, epi, seg, m0, n0, tn, wave, lane, stg, rows);
        } else {
          if (epi.a.part_dy) epilogue8_resid<false, true>(acc, epi, seg, m0, n0, tn, wave, lane, stg, rows);
          else epilogue8_resid<false, false>(acc, epi, seg, m0, n0, tn, wave, lane, stg, rows);
        }
        return;
      }
    }
    if constexpr (std::is_same<Epi, EpiF32>::value) {
      if (epi.vec && n0 + BN <= N) {
        epilogue8_f32(acc, epi, m0, n0, M, wave, lane, stg);
        return;
      }
    }
    epilogue8(acc, epi, m0, n0, M, N, tn, wave, lane, stg, rows);
  }
}

// ------------------------------------------------------------------ split forward's residual
// The forward product split over K leaves `parts` fp32 partial products
// [M, N] spaced part_stride apart.  One wave per (row m, 256-column tile):
// y = ((p0 + p1) + ...) + bias[m], then the residual epilogue's arithmetic
// (r = y - y_fp, dY = bf16(r * scale)) and the tile's sums of r^2 and of dY.
__global__ __launch_bounds__(256) void resid_parts_kernel(const float* __restrict__ P, int parts,
                                                          int64_t part_stride, int64_t M,
                                                          int64_t N, ResidArgs a, bool vec4) {
  const int lane = threadIdx.x & 63;
  const int64_t wid = (int64_t(blockIdx.x) * 256 + threadIdx.x) >> 6;
  if (wid >= M * a.ntn) return;                  // whole waves leave together
  const int64_t m = wid / a.ntn;
  const int tn = int(wid - m * a.ntn);
  const EpiResid<uint16_t> ep{a, false};
  const auto r = ep.row(m);
  const int64_t n0 = int64_t(tn) * BN + 4 * lane;
  float sq = 0.f, sdy = 0.f;
  if (vec4 && n0 + 4 <= N) {
    float4 y = *reinterpret_cast<const float4*>(P + m * N + n0);
    for (int q = 1; q < parts; ++q) {
      const float4 t = *reinterpret_cast<const float4*>(P + q * part_stride + m * N + n0);
      y.x += t.x;
      y.y += t.y;
      y.z += t.z;
      y.w += t.w;
    }
    const uint2 f = *reinterpret_cast<const uint2*>(r.yfp + n0);
    const float yv[4] = {y.x, y.y, y.z, y.w};
    const float fv[4] = {__uint_as_float(f.x << 16), __uint_as_float(f.x & 0xffff0000u),
                         __uint_as_float(f.y << 16), __uint_as_float(f.y & 0xffff0000u)};
    float d[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float res = (yv[e] + r.b) - fv[e];
      d[e] = res * r.scale;
      sq += res * res;
      sdy += EpiResid<uint16_t>::rounded(d[e]);
    }
    *reinterpret_cast<uint2*>(r.dy + n0) = make_uint2(f2bf2(d[0], d[1]), f2bf2(d[2], d[3]));
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t n = n0 + e;
      if (n < N) {
        float y = P[m * N + n];
        for (int q = 1; q < parts; ++q) y += P[q * part_stride + m * N + n];
        const float res = (y + r.b) - load1(r.yfp + n);
        const float d = res * r.scale;
        store1(r.dy + n, d);
        sq += res * res;
        sdy += EpiResid<uint16_t>::rounded(d);
      }
    }
  }
  sq = wave_sum(sq);
  sdy = wave_sum(sdy);
  if (lane == 0) ep.finish(m, tn, sq, sdy);
}

// ------------------------------------------------------------------ fp32 kernel
template <class Epi>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A,
                                                       const float* __restrict__ B, int64_t M,
                                                       int64_t N, int64_t K, int64_t lda,
                                                       int64_t ldb, Epi epi) {
  __shared__ float As[16][F32_TILE + 4];
  __shared__ float Bs[16][F32_TILE + 4];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int64_t m0 = int64_t(blockIdx.y) * F32_TILE, n0 = int64_t(blockIdx.x) * F32_TILE;
  const int lr = tid >> 2, lk = (tid & 3) * 4;
  float acc[4][4] = {};
  for (int64_t k0 = 0; k0 < K; k0 += 16) {
    const int64_t k = k0 + lk;
    float4 va = make_float4(0.f, 0.f, 0.f, 0.f), vb = va;
    if (m0 + lr < M && k < K) va = *reinterpret_cast<const float4*>(A + (m0 + lr) * lda + k);
    if (n0 + lr < N && k < K) vb = *reinterpret_cast<const float4*>(B + (n0 + lr) * ldb + k);
    As[lk + 0][lr] = va.x; As[lk + 1][lr] = va.y; As[lk + 2][lr] = va.z; As[lk + 3][lr] = va.w;
    Bs[lk + 0][lr] = vb.x; Bs[lk + 1][lr] = vb.y; Bs[lk + 2][lr] = vb.z; Bs[lk + 3][lr] = vb.w;
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t m = m0 + ty * 4 + i;
    float sq = 0.f, sdy = 0.f;
    if (m < M) {
      auto rowc = epi.row(m);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t n = n0 + tx * 4 + j;
        if (n < N) {
          float v1[8] = {acc[i][j], 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
          float2 c = epi.apply8(rowc, n, v1, 1);
          sq += c.x;
          sdy += c.y;
        }
      }
    }
    if constexpr (Epi::kRows) {
      sq = group_sum<16>(sq);
      sdy = group_sum<16>(sdy);
      if (tx == 0 && m < M) epi.finish(m, int(blockIdx.x), sq, sdy);
    }
  }
}

// The 8-wave kernel applies when K is a multiple of 64 and every operand
// offset of a tile fits the kernel's 32-bit byte offsets.
bool w8_ok(bool amn, bool bmn, int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldb) {
  if (K <= 0 || K % BK || lda % 8 || ldb % 8) return false;
  auto fits = [](bool mn, int64_t extent, int64_t ld) {
    return mn ? (extent >= 8 && extent % 8 == 0 && extent <= ld && ld < (int64_t(1) << 25))
              : ld < (int64_t(1) << 23);
  };
  return fits(amn, M, lda) && fits(bmn, N, ldb);
}

template <class Epi, bool AMN, bool BMN>
void launch_w8(const void* A, const void* B, int64_t M, int64_t N, int64_t K, int64_t lda,
               int64_t ldb, int64_t tm, int64_t tn, Epi epi, hipStream_t st, int splits = 1) {
  hipLaunchKernelGGL((gemm_bf16_w8_kernel<Epi, AMN, BMN>), dim3(unsigned(tm * tn * splits)),
                     dim3(NTHR8), 0,
                     st, static_cast<const uint16_t*>(A), static_cast<const uint16_t*>(B), M, N, K,
                     lda, ldb, int(tm), int(tn), epi);
}

// amn / bmn: operand stored MN-major (A as [K, M], B as [K, N]); bf16 only,
// fp32 output only, 8-wave kernel only.
template <class Epi>
hipError_t launch(const void* A, const void* B, bool bf16, int64_t M, int64_t N, int64_t K,
                  int64_t lda, int64_t ldb, Epi epi, hipStream_t st, bool amn = false,
                  bool bmn = false, int splits = 1) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (bf16) {
    const int64_t tm = (M + BM - 1) / BM, tn = (N + BN - 1) / BN;
    if (tm * tn * splits > (int64_t(1) << 31) - 1) return hipErrorInvalidValue;
    if (w8_ok(amn, bmn, M, N, K, lda, ldb)) {
      if (!amn && !bmn) {
        launch_w8<Epi, false, false>(A, B, M, N, K, lda, ldb, tm, tn, epi, st, splits);
      } else if constexpr (std::is_same<Epi, EpiF32>::value) {
        if (amn && bmn)
          launch_w8<Epi, true, true>(A, B, M, N, K, lda, ldb, tm, tn, epi, st, splits);
        else if (bmn)
          launch_w8<Epi, false, true>(A, B, M, N, K, lda, ldb, tm, tn, epi, st, splits);
        else
          launch_w8<Epi, true, false>(A, B, M, N, K, lda, ldb, tm, tn, epi, st, splits);
      } else {
        return hipErrorInvalidValue;
      }
    } else if (splits != 1) {
      return hipErrorInvalidValue;
    } else if (!amn && !bmn) {
      hipLaunchKernelGGL((gemm_bf16_kernel<Epi, false>), dim3(unsigned(tm * tn)), dim3(NTHR), 0,
                         st, static_cast<const uint16_t*>(A), static_cast<const uint16_t*>(B), M, N,
                         K, lda, ldb, int(tm), int(tn), epi);
    } else {
      return hipErrorInvalidValue;
    }
  } else {
    if (amn || bmn || splits != 1) return hipErrorInvalidValue;
    const int64_t tm = (M + F32_TILE - 1) / F32_TILE, tn = (N + F32_TILE - 1) / F32_TILE;
    if (tm > 65535 || tn > (int64_t(1) << 31) - 1) return hipErrorInvalidValue;
    hipLaunchKernelGGL(gemm_f32_kernel<Epi>, dim3(unsigned(tn), unsigned(tm)), dim3(256), 0, st,
                       static_cast<const float*>(A), static_cast<const float*>(B), M, N, K, lda,
                       ldb, epi);
  }
  return hipGetLastError();
}

}  // namespace

int gemm_part_tile_n(bool bf16) { return bf16 ? BN : F32_TILE; }

hipError_t gemm_nt_f32out(const void* A, const void* B, bool bf16, int64_t M, int64_t N,
                          int64_t K, int64_t lda, int64_t ldb, float* C, int64_t ldc,
                          hipStream_t st) {
  const bool vec = ldc % 8 == 0 && (reinterpret_cast<uintptr_t>(C) & 15) == 0;
  return launch(A, B, bf16, M, N, K, lda, ldb, EpiF32{C, ldc, vec}, st);
}

bool gemm_mn_supported(bool a_mn, bool b_mn, int64_t M, int64_t N, int64_t K, int64_t lda,
                       int64_t ldb) {
  return w8_ok(a_mn, b_mn, M, N, K, lda, ldb);
}

int gemm_mn_splits(bool a_mn, bool b_mn, int64_t M, int64_t N, int64_t K, int64_t lda,
                   int64_t ldb) {
  // Time in k-steps of one tile (a 256 x 256 x 64 MFMA step, ~1.65 us on a
  // loaded CU): whole waves of units, each K/(64 S) steps plus an fp32
  // epilogue worth ~16 steps, then the partial sum's (S + 1) M N 4 bytes at
  // ~5 TB/s.
  constexpr int kCUs = 256;
  constexpr double kStep = 1.65e-6, kEpi = 16.0, kBw = 5.0e12;
  const int64_t tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  int best = 1;
  double best_t = 0.0;
  for (int s = 1; s <= 8; s *= 2) {
    if (K % (int64_t(BK) * s)) break;
    const int64_t ks = K / s;
    if (s > 1 && (ks < 16 * BK || !w8_ok(a_mn, b_mn, M, N, ks, lda, ldb))) break;
    const int64_t waves = (tiles * s + kCUs - 1) / kCUs;
    double t_s = double(waves) * (double(ks / BK) + kEpi) * kStep;
    if (s > 1) t_s += double(s + 1) * double(M) * double(N) * 4.0 / kBw;
    if (s == 1 || t_s < 0.99 * best_t) {
      best = s;
      best_t = t_s;
    }
  }
  return best;
}

hipError_t gemm_f32out_mn(const void* A, bool a_mn, const void* B, bool b_mn, int64_t M,
                          int64_t N, int64_t K, int64_t lda, int64_t ldb, float* C, int64_t ldc,
                          hipStream_t st, int splits, int64_t split_stride) {
  if (splits < 1 || K % splits) return hipErrorInvalidValue;
  const int64_t ks = K / splits;
  if (splits > 1 && !w8_ok(a_mn, b_mn, M, N, ks, lda, ldb)) return hipErrorInvalidValue;
  const bool vec = ldc % 8 == 0 && (reinterpret_cast<uintptr_t>(C) & 15) == 0 &&
                   split_stride % 8 == 0;
  return launch(A, B, true, M, N, ks, lda, ldb, EpiF32{C, ldc, vec, split_stride}, st, a_mn,
                b_mn, splits);
}

bool gemm_wgrad_lwc_supported(int64_t M, int64_t C, int64_t K, int group) {
  return group >= 8 && group <= BN && (group & (group - 1)) == 0 && C % group == 0 &&
         w8_ok(false, true, M, C, K, K, C);
}

hipError_t gemm_wgrad_lwc(const void* dyT, const void* x, int64_t M, int64_t C, int64_t K,
                          int64_t lda, int64_t ldb, const LwcArgs& la, hipStream_t st) {
  if (!gemm_wgrad_lwc_supported(M, C, K, la.group) || lda != K || ldb != C || la.C != C ||
      la.ng != C / la.group || la.nseg < 1 || la.nseg > MAX_SEG)
    return hipErrorInvalidValue;
  auto go = [&](auto gc) {
    constexpr int Gc = decltype(gc)::value;
    const int64_t tm = (M + BM - 1) / BM, tn = (C + BN - 1) / BN;
    if (tm * tn > (int64_t(1) << 31) - 1) return hipErrorInvalidValue;
    launch_w8<EpiLwc<Gc>, false, true>(dyT, x, M, C, K, lda, ldb, tm, tn, EpiLwc<Gc>{la}, st);
    return hipGetLastError();
  };
  switch (la.group / 8) {
    case 1: return go(std::integral_constant<int, 1>{});
    case 2: return go(std::integral_constant<int, 2>{});
    case 4: return go(std::integral_constant<int, 4>{});
    case 8: return go(std::integral_constant<int, 8>{});
    case 16: return go(std::integral_constant<int, 16>{});
    default: return go(std::integral_constant<int, 32>{});
  }
}

hipError_t gemm_nt_store(const void* A, const void* B, bool bf16, int64_t M, int64_t N,
                         int64_t K, int64_t lda, int64_t ldb, void* C, bool c_bf16, int64_t ldc,
                         const float* bias, hipStream_t st) {
  const bool vec = ldc % 8 == 0 && (reinterpret_cast<uintptr_t>(C) & 15) == 0;
  if (c_bf16)
    return launch(A, B, bf16, M, N, K, lda, ldb,
                  EpiStore<uint16_t>{static_cast<uint16_t*>(C), ldc, bias, vec}, st);
  return launch(A, B, bf16, M, N, K, lda, ldb,
                EpiStore<float>{static_cast<float*>(C), ldc, bias, vec}, st);
}

int gemm_resid_splits(int64_t M, int64_t N, int64_t K) {
  // Same step model as gemm_mn_splits; the parts cost 2 S M N 4 bytes more
  // (written by the product, read by the residual pass).
  constexpr int kCUs = 256;
  constexpr double kStep = 1.45e-6, kEpi = 16.0, kBw = 5.0e12;
  if (!w8_ok(false, false, M, N, K, K, K)) return 1;
  const int64_t tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  int best = 1;
  double best_t = 0.0;
  for (int s = 1; s <= 4; s *= 2) {
    if (K % (int64_t(BK) * s)) break;
    const int64_t ks = K / s;
    if (s > 1 && ks < 16 * BK) break;
    const int64_t waves = (tiles * s + kCUs - 1) / kCUs;
    double t_s = double(waves) * (double(ks / BK) + kEpi) * kStep;
    if (s > 1) t_s += 2.0 * s * double(M) * double(N) * 4.0 / kBw + 5e-6;
    if (s == 1 || t_s < 0.9 * best_t) {
      best = s;
      best_t = t_s;
    }
  }
  return best;
}

hipError_t gemm_nt_resid_split(const void* A, const void* B, int64_t M, int64_t N, int64_t K,
                               int64_t lda, int64_t ldb, ResidArgs ra, float* parts, int splits,
                               hipStream_t st) {
  if (splits < 2 || K % splits || M <= 0 || N <= 0) return hipErrorInvalidValue;
  const int64_t ks = K / splits;
  if (!w8_ok(false, false, M, N, ks, lda, ldb)) return hipErrorInvalidValue;
  ra.ntn = int((N + BN - 1) / BN);
  const int64_t stride = M * N;
  const bool vec = N % 8 == 0 && (reinterpret_cast<uintptr_t>(parts) & 15) == 0;
  hipError_t e = launch(A, B, true, M, N, ks, lda, ldb, EpiF32{parts, N, vec, stride}, st, false,
                        false, splits);
  if (e != hipSuccess) return e;
  const int64_t waves = M * ra.ntn;
  // 16-byte part loads, 8-byte target loads and dY stores when every row allows them
  bool vec4 = N % 4 == 0 && ra.ld_yfp % 4 == 0 && ra.ld_dy % 4 == 0 &&
              (reinterpret_cast<uintptr_t>(ra.dy) & 7) == 0;
  for (int s = 0; s < ra.nseg; ++s) vec4 = vec4 && (reinterpret_cast<uintptr_t>(ra.yfp[s]) & 7) == 0;
  hipLaunchKernelGGL(resid_parts_kernel, dim3(unsigned((waves + 3) / 4)), dim3(256), 0, st, parts,
                     splits, stride, M, N, ra, vec4);
  return hipGetLastError();
}

hipError_t gemm_nt_resid(const void* A, const void* B, bool bf16, int64_t M, int64_t N,
                         int64_t K, int64_t lda, int64_t ldb, ResidArgs ra, hipStream_t st) {
  ra.ntn = int((N + gemm_part_tile_n(bf16) - 1) / gemm_part_tile_n(bf16));
  bool vec = ra.ld_yfp % 8 == 0 && ra.ld_dy % 8 == 0 &&
             (reinterpret_cast<uintptr_t>(ra.dy) & 15) == 0;
  for (int s = 0; s < ra.nseg; ++s) vec = vec && (reinterpret_cast<uintptr_t>(ra.yfp[s]) & 15) == 0;
  if (bf16) return launch(A, B, true, M, N, K, lda, ldb, EpiResid<uint16_t>{ra, vec}, st);
  return launch(A, B, false, M, N, K, lda, ldb, EpiResid<float>{ra, vec}, st);
}

}  // namespace oq
