// Host-visible argument structs and launchers of the MicroMix HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mm {

// Fused reorder-and-quantize of `rows` bf16 rows (activations or weights).
struct QuantArgs {
  const uint16_t* x;
  int64_t ldx;  // elements
  const int32_t* perm;
  int64_t rows;
  int K;
  int nb4, nb6;  // block counts of the E2M1 and E3M2 groups
  uint8_t* q4;
  int64_t ld4;
  uint8_t* q6;
  int64_t ld6;
  uint8_t* q8;
  int64_t ld8;
  uint8_t* sc;
  int64_t ldsc;
};

// One quantised GEMM operand.
struct Operand {
  const uint8_t* q[3];  // E2M1, E3M2, E4M3 code buffers
  int64_t ld[3];
  const uint8_t* sc;
  int64_t ldsc;
  int64_t rows;
};

struct GemmArgs {
  Operand w;  // first MFMA operand: weight rows (output columns n)
  Operand x;  // second MFMA operand: activation rows (output rows m)
  int nb[3];  // blocks per group
  uint16_t* y;
  int64_t ldy;
};

hipError_t launch_quantize(const QuantArgs& a, hipStream_t stream);
hipError_t launch_gemm_direct(const GemmArgs& a, hipStream_t stream);
hipError_t launch_gemm_tiled(const GemmArgs& a, hipStream_t stream);

}  // namespace mm
