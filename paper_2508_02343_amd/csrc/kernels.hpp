// Host-visible argument structs and launchers of the MicroMix HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mm {

// Packed-layout constants (the layout is documented in include/micromix.h).
constexpr int kRowGroup = 32;   // rows per row group
constexpr int kStepBlocks = 4;  // blocks per step
// Bytes of one row's step per group: E2M1, E3M2, E4M3.
__host__ __device__ constexpr int step_row_bytes(int group) { return group == 0 ? 64 : (group == 1 ? 96 : 128); }
// Bytes of one 32-element block per group.
__host__ __device__ constexpr int block_bytes(int group) { return group == 0 ? 16 : (group == 1 ? 24 : 32); }

// Byte offset, inside a group's code buffer, of block j (0..3) of step `step`
// of row n (row-group record, block-major): E2M1 16 bytes, E3M2 24 bytes,
// E4M3 the first 16 bytes (the second 16 are 512 bytes further on).
template <int G>
__host__ __device__ __forceinline__ int64_t code_offset(int64_t step, int64_t rp, int64_t n, int j) {
  constexpr int RB = step_row_bytes(G);
  const int64_t rec = (step * rp + (n & ~(int64_t)(kRowGroup - 1))) * RB;
  const int r = (int)(n & (kRowGroup - 1));
  if constexpr (G == 0) return rec + j * 512 + r * 16;
  else if constexpr (G == 1) return rec + j * 768 + r * 24;
  else return rec + (2 * j) * 512 + r * 16;
}

// Fused reorder-and-quantize of `rows` bf16 rows (activations or weights).
struct QuantArgs {
  const uint16_t* x;
  int64_t ldx;  // elements
  const int32_t* perm;
  int64_t rows;
  int64_t rp;    // rows rounded up to a row group
  int K;
  int nb[3];     // blocks per group
  int steps[3];  // steps per group
  uint8_t* q[3];
  uint8_t* sc;
  int fs;  // format set: bit 0 the 6-bit group is E2M3 (else E3M2), bit 1 the 8-bit group is E5M2 (else E4M3)
  // RMSNorm before the quantisation (norm != 0): x -> bf16(gamma * bf16(x * r)),
  // r = fp32(1 / sqrt(mean(x^2) + eps)) per row, gamma bf16 [K] in channel order
  int norm;
  const uint16_t* gamma;
  float eps;
};

// One quantised GEMM operand.
struct Operand {
  const uint8_t* q[3];  // E2M1, E3M2, E4M3 code buffers
  const uint8_t* sc;
  int64_t rows;
  int64_t rp;  // rows rounded up to a row group
};

struct GemmArgs {
  Operand w;     // first MFMA operand: weight rows (output columns n)
  Operand x;     // second MFMA operand: activation rows (output rows m)
  int steps[3];  // steps per group
  uint16_t* y;
  int64_t ldy;
  int fs;  // format set of both operands (as QuantArgs::fs)
};

// Offline calibration over X [rows, K]: channel sums in fixed row chunks,
// means, the stable order of the means, and the split.
constexpr int kCalibMaxWorkgroups = 256;  // column-sum workgroups at most (one per CU)
constexpr int kCalibSlice = 256;          // means per rank slice
struct CalibArgs {
  const uint16_t* x;
  int64_t ldx;  // elements
  int64_t rows;
  int K;
  int nchunks;         // row chunks of the column sums
  int64_t chunk_rows;  // rows per chunk (the last may be shorter)
  uint32_t* wgmax;     // [nmax] largest |x| of each column-sum workgroup, fp32 bit patterns
  int nmax;            // nchunks * tiles
  double* partial;     // [nchunks, K] per-chunk sums of |x|
  double* mean;        // [K]
  int32_t* slice_counts;  // [ceil(K / 256), K] channels of each 256-slice that sort before j
  int32_t* counts;     // [2 * ceil(K / 256)] G4 and G6 counts per 256-channel block
  int32_t* perm;       // [K] output sigma
  int32_t* split;      // [3] output (p4, p6, p8)
  int fp6_e2m3;        // T(6) with E2M3's constants instead of E3M2's
};

// Size of the library-owned calibration scratch (a static device array, one
// per GPU, held until the process ends) that mm_calibrate_no_alloc uses in
// place of a caller's workspace.  16 MiB covers every calibration plan up
// to K = 31488 channels, whatever the number of rows.
constexpr int64_t kCalibScratchBytes = 16ll << 20;

hipError_t launch_quantize(const QuantArgs& a, hipStream_t stream);
hipError_t launch_calibrate(const CalibArgs& a, hipStream_t stream);
// Device address of the current device's calibration scratch: looked up
// with hipGetSymbolAddress on the first call on each device, with that
// device current, and cached per device.  Allocates nothing.
hipError_t calibrate_scratch(void** ptr);
hipError_t launch_gemm_direct(const GemmArgs& a, hipStream_t stream);
hipError_t launch_gemm_tiled(const GemmArgs& a, hipStream_t stream);

}  // namespace mm
