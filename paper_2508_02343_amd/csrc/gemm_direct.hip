// Mixed MX GEMM for few activation rows (decode, M <= 64): memory-bound on the
// weight stream, so every lane loads its MFMA fragments straight from global
// memory (no LDS staging).  A workgroup covers a strip of R weight rows (the
// output's columns) so that the grid spans all CUs, and its four or eight
// wavefronts split the K loop between them and add their fp32 partial sums
// in LDS before the single bf16 rounding (Sec. 3.2 "GEMM kernel": fp32
// partials, bf16 out).  An output's summation order depends on the split, K
// and the number of wavefronts only, not on which strip holds it.
//
// Each wavefront works on the steps of one group only (the wavefronts are
// shared out between the groups by their numbers of steps), so the loads
// of all three groups are in flight at once instead of one group after the
// other; inside its group a wavefront issues the loads of several steps
// before the first of their MFMAs.  Per batch of steps, the E8M0 scales come
// as one 4-byte word per lane and tile (the four block scales of one row at
// one step) and reach the lanes that feed them to the MFMA through a
// cross-lane read, instead of one single-byte load per lane and step.
#include "gemm_common.hpp"

namespace mm {

// Steps a wavefront loads before their MFMAs: fewer for the widest tiles
// (eight or more 16 x 16 tiles: their fragments of one step take 64 or more
// registers).
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
// down.  Weight rows past the strip (R) or past N, and activation rows past
// the real ones, are not loaded (zero codes, unit scale): they only reach
// outputs that are never stored.  The weight is read once: its E2M1 and E4M3
// loads are non-temporal (N = 14336 E4M3: 12.7 -> 11.9 us).
template <int TN, int TM, int G, int FS>
__device__ __forceinline__ void direct_group(const GemmArgs& a, v4f (&acc)[TN][TM], int64_t n0, int R, int64_t m0,
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
        const int64_t n = n0 + 16 * i + r;
        wsw[i] = sval && 16 * i + r < R && n < a.w.rows ? load_scale_word(a.w.sc, a.w.rp, t0 + su, n) : 0x7f7f7f7fu;
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
          const int64_t n = n0 + 16 * i + r;
          wf[u][i] = 16 * i + r < R && n < a.w.rows ? load_frag16_global<G, true>(a.w.q[G], a.w.rp, n, s, g)
                                                     : v8i{0, 0, 0, 0, 0, 0, 0, 0};
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

// Workgroup b covers weight rows [b R, b R + R) in TN tiles of 16 (rows
// past R or N not loaded, not stored).  Wavefronts [0, w0) work on group 0,
// [w0, w0 + w1) on group 1, the next w2 on group 2; the partial sums are
// added in wavefront order, wavefront t adding up tiles t, t + W, ...
template <int TN, int TM, int W, int FS>
__global__ __launch_bounds__(64 * W) void gemm_direct_kernel(GemmArgs a, int R, int w0, int w1, int w2) {
  __shared__ v4f red[W][TN * TM][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t n0 = (int64_t)blockIdx.x * R;
  const int64_t m0 = (int64_t)blockIdx.y * (16 * TM);

  v4f acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  if (wave < w0) direct_group<TN, TM, 0, FS>(a, acc, n0, R, m0, wave, w0, lane);
  else if (wave < w0 + w1) direct_group<TN, TM, 1, FS>(a, acc, n0, R, m0, wave - w0, w1, lane);
  else if (wave < w0 + w1 + w2) direct_group<TN, TM, 2, FS>(a, acc, n0, R, m0, wave - w0 - w1, w2, lane);

#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) red[wave][i * TM + j][lane] = acc[i][j];
  __syncthreads();
  const int g = lane >> 4, r = lane & 15;
  const int64_t nend = n0 + R < a.w.rows ? n0 + R : a.w.rows;
  for (int t = wave; t < TN * TM; t += W) {
    if (16 * (t / TM) >= R) continue;  // a tile wholly past the workgroup's rows
    v4f c = red[0][t][lane];
#pragma unroll
    for (int w = 1; w < W; ++w) c += red[w][t][lane];
    store_out4(a, m0 + 16 * (t % TM) + r, n0 + 16 * (t / TM) + 4 * g, c, a.x.rows, nend);
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
static hipError_t launch_direct_fs(const GemmArgs& a, int R, hipStream_t stream) {
  const dim3 grid((unsigned)((a.w.rows + R - 1) / R), (unsigned)((a.x.rows + 16 * TM - 1) / (16 * TM)));
  int w[3];
  direct_waves(a, W, w);
  hipLaunchKernelGGL((gemm_direct_kernel<TN, TM, W, FS>), grid, dim3(64 * W), 0, stream, a, R, w[0], w[1], w[2]);
  return hipGetLastError();
}

// The format set is an instruction immediate: one kernel per set.
template <int TN, int TM, int W>
static hipError_t launch_direct(const GemmArgs& a, int R, hipStream_t stream) {
  switch (a.fs) {
    case 0: return launch_direct_fs<TN, TM, W, 0>(a, R, stream);
    case 1: return launch_direct_fs<TN, TM, W, 1>(a, R, stream);
    case 2: return launch_direct_fs<TN, TM, W, 2>(a, R, stream);
    case 3: return launch_direct_fs<TN, TM, W, 3>(a, R, stream);
    default: return hipErrorInvalidValue;
  }
}

template <int TM>
static hipError_t launch_direct_tm(const GemmArgs& a, int R, hipStream_t stream) {
  if (R <= 16) return launch_direct<1, TM, 8>(a, R, stream);
  if (R <= 32) return launch_direct<2, TM, 8>(a, R, stream);
  return launch_direct<4, TM, 8>(a, R, stream);
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

// Rows per workgroup for two or more activation tiles: the fewest multiple
// of 8 (at least 16, at most 64) that spreads the weight rows evenly over k
// workgroups per CU, k as small as that allows, so that every CU streams
// about the same number of bytes and each activation fragment feeds up to
// four weight tiles.
static int direct_rows(int64_t N, int cus) {
  int64_t k = N / (64 * (int64_t)cus);
  for (k = k < 1 ? 1 : k;; ++k) {
    int64_t R = (N + k * cus - 1) / (k * cus);
    R = (R + 7) / 8 * 8;
    if (R <= 64) return R < 16 ? 16 : (int)R;
  }
}

// One activation tile (M <= 16): a whole 32-row group per workgroup (each
// step's loads are one contiguous 2 KB record) with four wavefronts when that
// still gives every CU a strip, else 16-row strips with eight wavefronts.
// Measured against the even spread above on this tile: 7.7 against 8.3 us
// (N = 14336, E2M1), equal for E4M3.
hipError_t launch_gemm_direct(const GemmArgs& a, hipStream_t stream) {
  int cus = 0;
  hipError_t e = direct_cus(&cus);
  if (e != hipSuccess) return e;
  const int64_t M = a.x.rows;
  if (M <= 16) {
    if ((a.w.rows + 31) / 32 >= cus) return launch_direct<2, 1, 4>(a, 32, stream);
    return launch_direct<1, 1, 8>(a, 16, stream);
  }
  const int R = direct_rows(a.w.rows, cus);
  return M <= 32 ? launch_direct_tm<2>(a, R, stream) : launch_direct_tm<4>(a, R, stream);
}

}  // namespace mm
