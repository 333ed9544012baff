// Mixed MX GEMM for few activation rows (decode, M <= 64): memory-bound on the
// weight stream, so every lane loads its MFMA fragments straight from global
// memory (no LDS staging), a workgroup covers a narrow strip of output
// columns so that the grid spans all CUs, and the workgroup's four or eight
// wavefronts split the K loop between them and add their fp32 partial sums
// in LDS before the single bf16 rounding (Sec. 3.2 "GEMM kernel": fp32
// partials, bf16 out).  Each wavefront issues the loads of several of its
// steps of a group before the first of their MFMAs, so it has that many
// steps of weight in flight instead of a chain of one load, then one MFMA,
// per step.
#include "gemm_common.hpp"

namespace mm {

// Steps a wavefront loads before their MFMAs: fewer for the widest tile
// (its fragments of one step already take 54 registers).
template <int TN, int TM>
__host__ __device__ constexpr int direct_batch() { return TN * TM >= 8 ? 2 : 4; }

// Group G's layout steps: wavefront w of W takes steps w, w + W, ..., U at
// a time, issuing all U steps' loads before the first of their MFMAs.
template <int TN, int TM, int W, int G, int FS>
__device__ __forceinline__ void direct_group(const GemmArgs& a, v4f (&acc)[TN][TM], int64_t n0, int64_t m0,
                                             int wave, int lane) {
  constexpr int U = direct_batch<TN, TM>();
  const int S = a.steps[G];
  if (S == 0) return;
  const int g = lane >> 4, r = lane & 15;
  // global step index of this group's first step inside the scale buffer
  const int t0 = (G >= 1 ? a.steps[0] : 0) + (G >= 2 ? a.steps[1] : 0);
  for (int s0 = wave; s0 < S; s0 += W * U) {
    v8i wf[U][TN], xf[U][TM];
    int ws[U][TN], xs[U][TM];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = s0 + W * u;
      if (s < S) {  // uniform over the wavefront
#pragma unroll
        for (int i = 0; i < TN; ++i) {
          int64_t n = n0 + 16 * i + r;
          n = n < a.w.rp ? n : a.w.rp - 1;  // padded rows exist up to rp
          wf[u][i] = load_frag16_global<G>(a.w.q[G], a.w.rp, n, s, g);
          ws[u][i] = load_scale(a.w.sc, a.w.rp, t0 + s, n, g);
        }
#pragma unroll
        for (int j = 0; j < TM; ++j) {
          int64_t m = m0 + 16 * j + r;
          m = m < a.x.rp ? m : a.x.rp - 1;
          xf[u][j] = load_frag16_global<G>(a.x.q[G], a.x.rp, m, s, g);
          xs[u][j] = load_scale(a.x.sc, a.x.rp, t0 + s, m, g);
        }
      }
    }
    // all of the batch's loads are issued before its first MFMA
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      // a step past the group's last (not loaded) adds exactly zero: zero
      // codes (+0 in every element format) under the unit scale
      const bool valid = s0 + W * u < S;
#pragma unroll
      for (int i = 0; i < TN; ++i) {
#pragma unroll
        for (int e = 0; e < 8; ++e) wf[u][i][e] = valid ? wf[u][i][e] : 0;
        ws[u][i] = valid ? ws[u][i] : 127;
      }
#pragma unroll
      for (int j = 0; j < TM; ++j) {
#pragma unroll
        for (int e = 0; e < 8; ++e) xf[u][j][e] = valid ? xf[u][j][e] : 0;
        xs[u][j] = valid ? xs[u][j] : 127;
      }
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j) MM_MFMA_GROUP(G, FS, acc[i][j], wf[u][i], xf[u][j], ws[u][i], xs[u][j]);
    }
  }
}

template <int TN, int TM, int W, int FS>
__global__ __launch_bounds__(64 * W) void gemm_direct_kernel(GemmArgs a) {
  __shared__ float red[W - 1][TN * TM * 4][64];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t n0 = (int64_t)blockIdx.x * (16 * TN);
  const int64_t m0 = (int64_t)blockIdx.y * (16 * TM);

  v4f acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  direct_group<TN, TM, W, 0, FS>(a, acc, n0, m0, wave, lane);
  direct_group<TN, TM, W, 1, FS>(a, acc, n0, m0, wave, lane);
  direct_group<TN, TM, W, 2, FS>(a, acc, n0, m0, wave, lane);

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
      for (int w = 0; w < W - 1; ++w)
#pragma unroll
        for (int q = 0; q < 4; ++q) c[q] += red[w][(i * TM + j) * 4 + q][lane];
      store_out4(a, m0 + 16 * j + r, n0 + 16 * i + 4 * g, c, a.x.rows, a.w.rows);
    }
}

template <int TN, int TM, int W, int FS>
static hipError_t launch_direct_fs(const GemmArgs& a, hipStream_t stream) {
  const dim3 grid((unsigned)((a.w.rows + 16 * TN - 1) / (16 * TN)), (unsigned)((a.x.rows + 16 * TM - 1) / (16 * TM)));
  hipLaunchKernelGGL((gemm_direct_kernel<TN, TM, W, FS>), grid, dim3(64 * W), 0, stream, a);
  return hipGetLastError();
}

// The format set is an instruction immediate: one kernel per set.
template <int TN, int TM, int W>
static hipError_t launch_direct(const GemmArgs& a, hipStream_t stream) {
  switch (a.fs) {
    case 0: return launch_direct_fs<TN, TM, W, 0>(a, stream);
    case 1: return launch_direct_fs<TN, TM, W, 1>(a, stream);
    case 2: return launch_direct_fs<TN, TM, W, 2>(a, stream);
    case 3: return launch_direct_fs<TN, TM, W, 3>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

// CUs of the current device (cached per thread for the last device).
static hipError_t direct_cus(int* cus) {
  thread_local int last_dev = -1, last_cus = 0;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev != last_dev) {
    e = hipDeviceGetAttribute(&last_cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    last_dev = dev;
  }
  *cus = last_cus;
  return hipSuccess;
}

// Output strips: a whole 32-row group of weight rows per workgroup (its
// loads are the group's contiguous 512-byte runs) when that still gives
// every CU a strip, with four wavefronts; else 16 rows per workgroup and
// eight wavefronts (twice the strips, half the steps per wavefront).
hipError_t launch_gemm_direct(const GemmArgs& a, hipStream_t stream) {
  int cus = 0;
  hipError_t e = direct_cus(&cus);
  if (e != hipSuccess) return e;
  const int64_t M = a.x.rows;
  const bool wide = (a.w.rows + 31) / 32 >= cus;
  if (M > 32) return launch_direct<2, 4, 4>(a, stream);
  if (wide) return M <= 16 ? launch_direct<2, 1, 4>(a, stream) : launch_direct<2, 2, 4>(a, stream);
  return M <= 16 ? launch_direct<1, 1, 8>(a, stream) : launch_direct<1, 2, 8>(a, stream);
}

}  // namespace mm
