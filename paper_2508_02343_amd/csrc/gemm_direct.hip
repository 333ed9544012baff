// Mixed MX GEMM for few activation rows (decode, M <= 64): memory-bound on the
// weight stream, so every lane loads its MFMA fragments straight from global
// memory (no LDS staging), a workgroup covers a narrow strip of output
// columns so that the grid spans all CUs, and the workgroup's four or eight
// wavefronts split the K loop between them and add their fp32 partial sums
// in LDS before the single bf16 rounding (Sec. 3.2 "GEMM kernel": fp32
// partials, bf16 out).
//
// Each wavefront works on the steps of one group only (the wavefronts are
// shared out between the groups in proportion to their steps), so the loads
// of all three groups are in flight at once instead of one group after the
// other; inside its group a wavefront issues the loads of several steps
// before the first of their MFMAs.  Per batch of steps, the E8M0 scales come
// as one 4-byte word per lane and tile (the four block scales of one row at
// one step) and reach the lanes that feed them to the MFMA through a
// cross-lane read, instead of one single-byte load per lane and step.
#include "gemm_common.hpp"

namespace mm {

// Steps a wavefront loads before their MFMAs: fewer for the widest tile
// (its fragments of one step already take 54 registers).
template <int TN, int TM>
__host__ __device__ constexpr int direct_batch() { return TN * TM >= 8 ? 2 : 4; }

// The four E8M0 block scales of row n at global step t: one 4-byte word
// (scale byte of block j at (t * rp + n) * 4 + j).
__device__ __forceinline__ uint32_t load_scale_word(const uint8_t* sc, int64_t rp, int64_t t, int64_t n) {
  return *(const __attribute__((address_space(1))) uint32_t*)(sc + (t * rp + n) * kStepBlocks);
}

// Group G's layout steps on the W wavefronts given to the group: wavefront
// w takes steps w, w + W, ..., U at a time, all U steps' loads issued before
// the first of their MFMAs.  Scale words: lane 16 u + r loads row r's word of
// step u of the batch; the lane (block b, row r) that the MFMA of step u
// takes the scale from reads that word from lane 16 u + r and shifts byte b
// down.  Activation rows past the real ones are not loaded (zero codes, unit
// scale): they only reach output rows that are never stored.
template <int TN, int TM, int G, int FS>
__device__ __forceinline__ void direct_group(const GemmArgs& a, v4f (&acc)[TN][TM], int64_t n0, int64_t m0,
                                             int wave, int W, int lane) {
  constexpr int U = direct_batch<TN, TM>();
  static_assert(U <= 4, "one scale word per lane holds the scales of four steps");
  const int S = a.steps[G];
  const int g = lane >> 4, r = lane & 15;
  // global step index of this group's first step inside the scale buffer
  const int t0 = (G >= 1 ? a.steps[0] : 0) + (G >= 2 ? a.steps[1] : 0);
  for (int s0 = wave; s0 < S; s0 += W * U) {
    v8i wf[U][TN], xf[U][TM];
    uint32_t wsw[TN], xsw[TM];
    {
      const int su = s0 + W * g;  // step of this lane's scale words
      const bool sval = g < U && su < S;
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        int64_t n = n0 + 16 * i + r;
        n = n < a.w.rp ? n : a.w.rp - 1;  // padded rows exist up to rp
        wsw[i] = sval ? load_scale_word(a.w.sc, a.w.rp, t0 + su, n) : 0x7f7f7f7fu;
      }
#pragma unroll
      for (int j = 0; j < TM; ++j) {
        const int64_t m = m0 + 16 * j + r;
        xsw[j] = sval && m < a.x.rows ? load_scale_word(a.x.sc, a.x.rp, t0 + su, m) : 0x7f7f7f7fu;
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = s0 + W * u;
      if (s < S) {  // uniform over the wavefront
#pragma unroll
        for (int i = 0; i < TN; ++i) {
          int64_t n = n0 + 16 * i + r;
          n = n < a.w.rp ? n : a.w.rp - 1;
          wf[u][i] = load_frag16_global<G>(a.w.q[G], a.w.rp, n, s, g);
        }
#pragma unroll
        for (int j = 0; j < TM; ++j) {
          const int64_t m = m0 + 16 * j + r;
          xf[u][j] = m < a.x.rows ? load_frag16_global<G>(a.x.q[G], a.x.rp, m, s, g) : v8i{0, 0, 0, 0, 0, 0, 0, 0};
        }
      }
    }
    // all of the batch's loads are issued before its first MFMA
    __builtin_amdgcn_sched_barrier(0);
    int ws[U][TN], xs[U][TM];
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int i = 0; i < TN; ++i) ws[u][i] = __builtin_amdgcn_ds_bpermute((16 * u + r) * 4, (int)wsw[i]);
#pragma unroll
      for (int j = 0; j < TM; ++j) xs[u][j] = __builtin_amdgcn_ds_bpermute((16 * u + r) * 4, (int)xsw[j]);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (s0 + W * u >= S) break;  // uniform: steps past the group's last were not loaded
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j)
          MM_MFMA_GROUP(G, FS, acc[i][j], wf[u][i], xf[u][j], (int)((uint32_t)ws[u][i] >> (8 * g)),
                        (int)((uint32_t)xs[u][j] >> (8 * g)));
    }
  }
}

// Wavefronts [0, w0) work on group 0, [w0, w0 + w1) on group 1, the next w2
// on group 2; the partial sums are added in wavefront order.
template <int TN, int TM, int W, int FS>
__global__ __launch_bounds__(64 * W) void gemm_direct_kernel(GemmArgs a, int w0, int w1, int w2) {
  __shared__ v4f red[W - 1][TN * TM][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t n0 = (int64_t)blockIdx.x * (16 * TN);
  const int64_t m0 = (int64_t)blockIdx.y * (16 * TM);

  v4f acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  if (wave < w0) direct_group<TN, TM, 0, FS>(a, acc, n0, m0, wave, w0, lane);
  else if (wave < w0 + w1) direct_group<TN, TM, 1, FS>(a, acc, n0, m0, wave - w0, w1, lane);
  else if (wave < w0 + w1 + w2) direct_group<TN, TM, 2, FS>(a, acc, n0, m0, wave - w0 - w1, w2, lane);

  if (wave > 0) {
#pragma unroll
    for (int i = 0; i < TN; ++i)
#pragma unroll
      for (int j = 0; j < TM; ++j) red[wave - 1][i * TM + j][lane] = acc[i][j];
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
      for (int w = 0; w < W - 1; ++w) c += red[w][i * TM + j][lane];
      store_out4(a, m0 + 16 * j + r, n0 + 16 * i + 4 * g, c, a.x.rows, a.w.rows);
    }
}

// Wavefronts per group: one for each group that has steps, then one at a
// time to the group whose wavefronts take the most steps each (ties: the
// wider format), so the longest chain of steps is as short as it can be.
static void direct_waves(const GemmArgs& a, int W, int* w) {
  const int* S = a.steps;
  for (int G = 0; G < 3; ++G) w[G] = S[G] > 0 ? 1 : 0;
  for (int k = w[0] + w[1] + w[2]; k < W && k > 0; ++k) {
    int best = -1, most = -1;
    for (int G = 2; G >= 0; --G) {
      if (w[G] == 0) continue;
      const int c = (S[G] + w[G] - 1) / w[G];
      if (c > most) {
        most = c;
        best = G;
      }
    }
    ++w[best];
  }
}

template <int TN, int TM, int W, int FS>
static hipError_t launch_direct_fs(const GemmArgs& a, hipStream_t stream) {
  const dim3 grid((unsigned)((a.w.rows + 16 * TN - 1) / (16 * TN)), (unsigned)((a.x.rows + 16 * TM - 1) / (16 * TM)));
  int w[3];
  direct_waves(a, W, w);
  hipLaunchKernelGGL((gemm_direct_kernel<TN, TM, W, FS>), grid, dim3(64 * W), 0, stream, a, w[0], w[1], w[2]);
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
