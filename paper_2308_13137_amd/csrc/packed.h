// Host-side launchers of the deployment kernels (packed low-bit weights and the
// weight-only quantised linear of Sec. 4.5), shared with the C ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace oq {

// Event-timing kind of the packed linear; it follows the kinds of ProfKind.
constexpr int PK_PACKED_LINEAR = 9;

// Largest input width the packed linear takes (one token's staged row must fit LDS).
constexpr int64_t PACKED_MAX_C_IN = 65536;

// codes [c_out, c_in] u8 -> packed [c_out, c_in * bits / 8]: each row one
// little-endian bit string (code j at bits j*bits ..).  c_in % 32 == 0.
hipError_t pack_codes(const uint8_t* codes, int64_t c_out, int64_t c_in, int bits,
                      uint8_t* packed, hipStream_t stream);

// Y[t, o] = sum_c X[t, c] * (q[o, c] - z[o, g]) * h[o, g] (+ bias[o]), g = c / group.
// X bf16 [n_tok, c_in]; Y [n_tok, c_out] fp32 or bf16; bits 2..7.
hipError_t packed_linear(const uint16_t* X, int64_t n_tok, int64_t c_in, const uint8_t* packed,
                         int bits, int64_t group, const float* h, const float* z,
                         const float* bias, int64_t c_out, void* Y, bool y_bf16,
                         hipStream_t stream);

}  // namespace oq
