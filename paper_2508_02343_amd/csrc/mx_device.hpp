// Element-format selectors shared by the MicroMix HIP kernels (gfx950 only).
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

}  // namespace mm
