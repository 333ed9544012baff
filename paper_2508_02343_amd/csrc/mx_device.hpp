// Device-side helpers shared by the MicroMix HIP kernels (gfx950 only).
//
// Element formats are the OCP MX ones the method uses (paper Appendix B,
// Table "tab:microscaling"; Sec. 4.1 "Quantization"): E2M1 for the MXFP4
// group, E3M2 for MXFP6 and E4M3 for MXFP8.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mm {

// Format selector values of the gfx950 block-scaled MFMA (cbsz / blgp).
enum MfmaFmt : int { kE4M3 = 0, kE5M2 = 1, kE2M3 = 2, kE3M2 = 3, kE2M1 = 4 };

// Per-format constants used by the encoder.
struct FmtParams {
  int mbits;   // mantissa bits
  int emin;    // exponent of the lowest binade (1 - bias)
  int emax;    // exponent of the top binade holding finite values
  int maxmag;  // largest finite code magnitude (sign bit clear)
  int bits;    // code width
};

__host__ __device__ constexpr FmtParams fmt_params(int group) {
  // group 0 = MXFP4 (E2M1), 1 = MXFP6 (E3M2), 2 = MXFP8 (E4M3)
  return group == 0   ? FmtParams{1, 0, 2, 0x7, 4}
         : group == 1 ? FmtParams{2, -2, 4, 0x1F, 6}
                      : FmtParams{3, -6, 8, 0x7E, 8};
}

// floor(log2 |x|) of a non-zero bf16 magnitude (15 bits, sign removed).
__device__ __forceinline__ int bf16_floor_log2(uint32_t mag) {
  const int E = (int)(mag >> 7);
  if (E) return E - 127;
  return (31 - __builtin_clz(mag & 0x7Fu)) - 133;  // subnormal: m * 2^-133
}

// Shared-scale exponent of a block from its largest bf16 magnitude:
// floor(log2 amax) - emax, clamped to the E8M0 range; -127 for a zero block.
__device__ __forceinline__ int block_exponent(uint32_t amax_mag, int emax) {
  if (amax_mag == 0) return -127;
  int e = bf16_floor_log2(amax_mag) - emax;
  return e < -127 ? -127 : (e > 127 ? 127 : e);
}

// Code of one bf16 element h under block exponent e: |x| * 2^-e rounded to
// the nearest representable magnitude (ties to even), saturated at the
// largest finite code, sign of x kept.  Pure integer arithmetic: the bf16
// significand is sig * 2^ex with sig < 2^8, and every grid point of the
// target format is n * 2^qe for an integer n, so rounding is a right shift
// of sig with round-half-even on the shifted-out bits.
__device__ __forceinline__ uint32_t encode_bf16(uint32_t h, int e, const FmtParams& f) {
  const uint32_t sign = (h >> 15) & 1u;
  const uint32_t mag = h & 0x7FFFu;
  const int E = (int)(mag >> 7);
  const int sig = E ? (int)((mag & 0x7Fu) | 0x80u) : (int)(mag & 0x7Fu);
  uint32_t code = 0;
  if (sig) {
    const int ex = (E ? E : 1) - 134 - e;         // value / 2^e = sig * 2^ex
    const int t = (31 - __builtin_clz(sig)) + ex;  // floor(log2 |x / 2^e|)
    const int tb = t > f.emin ? t : f.emin;        // binade used for the grid
    const int sh = (tb - f.mbits) - ex;            // sig >> sh gives the grid count
    int n;
    if (sh <= 0) {
      n = sig << (-sh);
    } else if (sh >= 9) {
      n = 0;  // sig < 2^8 < 2^(sh-1): below half a grid step
    } else {
      n = sig >> sh;
      const int rem = sig & ((1 << sh) - 1);
      const int half = 1 << (sh - 1);
      n += (rem > half) | ((rem == half) & (n & 1));
    }
    int c = ((tb - f.emin) << f.mbits) + n;
    code = (uint32_t)(c < f.maxmag ? c : f.maxmag);
  }
  return code | (sign << (f.bits - 1));
}

}  // namespace mm
