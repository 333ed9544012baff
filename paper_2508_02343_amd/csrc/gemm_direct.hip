// Mixed MX GEMM for few activation rows (decode, M <= 64): memory-bound on the
// weight stream, so every lane loads its MFMA fragments straight from global
// memory (no LDS staging), a workgroup covers a narrow strip of output
// columns so that the grid spans all CUs, and the workgroup's four wavefronts
// split the K loop between them and add their fp32 partial sums in LDS before
// the single bf16 rounding (Sec. 3.2 "GEMM kernel": fp32 partials, bf16 out).
#include "gemm_common.hpp"

namespace mm {

constexpr int kDirectWaves = 4;

template <int TN, int TM, int G, int FS>
__device__ __forceinline__ void direct_group(const GemmArgs& a, v4f (&acc)[TN][TM], int64_t n0, int64_t m0,
                                             int wave, int lane) {
  const int S = a.steps[G];
  if (S == 0) return;
  const int g = lane >> 4, r = lane & 15;
  // global step index of this group's first step inside the scale buffer
  const int t0 = (G >= 1 ? a.steps[0] : 0) + (G >= 2 ? a.steps[1] : 0);
  for (int s = wave; s < S; s += kDirectWaves) {
    v8i wf[TN], xf[TM];
    int ws[TN], xs[TM];
#pragma unroll
    for (int i = 0; i < TN; ++i) {
      int64_t n = n0 + 16 * i + r;
      n = n < a.w.rp ? n : a.w.rp - 1;  // padded rows exist up to rp
      wf[i] = load_frag16_global<G>(a.w.q[G], a.w.rp, n, s, g);
      ws[i] = load_scale(a.w.sc, a.w.rp, t0 + s, n, g);
    }
#pragma unroll
    for (int j = 0; j < TM; ++j) {
      int64_t m = m0 + 16 * j + r;
      m = m < a.x.rp ? m : a.x.rp - 1;
      xf[j] = load_frag16_global<G>(a.x.q[G], a.x.rp, m, s, g);
      xs[j] = load_scale(a.x.sc, a.x.rp, t0 + s, m, g);
    }
#pragma unroll
    for (int i = 0; i < TN; ++i)
#pragma unroll
      for (int j = 0; j < TM; ++j) MM_MFMA_GROUP(G, FS, acc[i][j], wf[i], xf[j], ws[i], xs[j]);
  }
}

template <int TN, int TM, int FS>
__global__ __launch_bounds__(64 * kDirectWaves) void gemm_direct_kernel(GemmArgs a) {
  __shared__ float red[kDirectWaves - 1][TN * TM * 4][64];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t n0 = (int64_t)blockIdx.x * (16 * TN);
  const int64_t m0 = (int64_t)blockIdx.y * (16 * TM);

  v4f acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  direct_group<TN, TM, 0, FS>(a, acc, n0, m0, wave, lane);
  direct_group<TN, TM, 1, FS>(a, acc, n0, m0, wave, lane);
  direct_group<TN, TM, 2, FS>(a, acc, n0, m0, wave, lane);

  if (wave > 0) {
#pragma unroll
    for (int i = 0; i < TN; ++i)
#pragma unroll
      for (int j = 0; j < TM; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) red[wave - 1][(i * TM + j) * 4 + q][lane] = acc[i][j][q];
  }
  __syncthreads();
  if (wave != 0) return;
  const int g = lane >> 4, r = lane & 15;
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) {
      v4f c = acc[i][j];
#pragma unroll
      for (int w = 0; w < kDirectWaves - 1; ++w)
#pragma unroll
        for (int q = 0; q < 4; ++q) c[q] += red[w][(i * TM + j) * 4 + q][lane];
      store_out4(a, m0 + 16 * j + r, n0 + 16 * i + 4 * g, c, a.x.rows, a.w.rows);
    }
}

template <int TN, int TM, int FS>
static hipError_t launch_direct_fs(const GemmArgs& a, hipStream_t stream) {
  const dim3 grid((unsigned)((a.w.rows + 16 * TN - 1) / (16 * TN)), (unsigned)((a.x.rows + 16 * TM - 1) / (16 * TM)));
  hipLaunchKernelGGL((gemm_direct_kernel<TN, TM, FS>), grid, dim3(64 * kDirectWaves), 0, stream, a);
  return hipGetLastError();
}

// The format set is an instruction immediate: one kernel per set.
template <int TN, int TM>
static hipError_t launch_direct(const GemmArgs& a, hipStream_t stream) {
  switch (a.fs) {
    case 0: return launch_direct_fs<TN, TM, 0>(a, stream);
    case 1: return launch_direct_fs<TN, TM, 1>(a, stream);
    case 2: return launch_direct_fs<TN, TM, 2>(a, stream);
    case 3: return launch_direct_fs<TN, TM, 3>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm_direct(const GemmArgs& a, hipStream_t stream) {
  const int64_t M = a.x.rows;
  if (M <= 16) return launch_direct<1, 1>(a, stream);
  if (M <= 32) return launch_direct<1, 2>(a, stream);
  return launch_direct<2, 4>(a, stream);
}

}  // namespace mm
