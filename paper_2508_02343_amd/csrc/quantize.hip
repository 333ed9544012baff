// Fused reorder-and-quantize (MicroMix Sec. 3.2 "Quantization kernel",
// Fig. "micromix-design" b): one pass over bf16 rows that gathers channels by
// sigma (Sec. 3.1), takes each 32-channel block's shared E8M0 scale and writes
// E2M1 / E3M2 / E4M3 codes for the three groups (Sec. 2.1 MX rule).
//
// Memory-bound design for gfx950:
//  - a workgroup owns R consecutive rows; the rows are streamed into LDS with
//    16-byte coalesced loads (the only HBM read);
//  - each thread owns a fixed run of 16 permuted channels (half a block) and
//    keeps its 16 sigma entries in registers for all R rows, so sigma is read
//    once per workgroup;
//  - the gather is a read from LDS; the block absmax is a max over the
//    thread's 16 values and one cross-lane exchange with the neighbour lane
//    that owns the other half of the block;
//  - codes are packed in registers and written with one 8-, 12- or 16-byte
//    store per thread, so a wavefront writes a contiguous span of each group.
#include "kernels.hpp"
#include "mx_device.hpp"

namespace mm {

__global__ __launch_bounds__(1024) void quantize_rows_kernel(QuantArgs a, int R) {
  extern __shared__ uint16_t lds_rows[];  // [R][K]
  const int tid = threadIdx.x;
  const int T = blockDim.x;
  const int64_t row0 = (int64_t)blockIdx.x * R;
  const int K = a.K;
  const int nrows = (int)((a.rows - row0) < R ? (a.rows - row0) : R);

  // 1. stream the rows into LDS (16 B per load, fully coalesced)
  const int chunks_per_row = K >> 3;
  const int total_chunks = nrows * chunks_per_row;
  for (int c = tid; c < total_chunks; c += T) {
    const int r = c / chunks_per_row;
    const int j = c - r * chunks_per_row;
    const uint4 v = *reinterpret_cast<const uint4*>(a.x + (row0 + r) * a.ldx + (int64_t)j * 8);
    *reinterpret_cast<uint4*>(lds_rows + r * K + j * 8) = v;
  }
  __syncthreads();

  // 2. every thread handles 16 permuted channels per row
  const int units = K >> 4;
  for (int u = tid; u < units; u += T) {
    int p[16];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int4 v = *reinterpret_cast<const int4*>(a.perm + u * 16 + q * 4);
      p[4 * q + 0] = v.x;
      p[4 * q + 1] = v.y;
      p[4 * q + 2] = v.z;
      p[4 * q + 3] = v.w;
    }
    // an out-of-range entry (a caller error) must not read outside the row
#pragma unroll
    for (int i = 0; i < 16; ++i) p[i] = (unsigned)p[i] < (unsigned)K ? p[i] : 0;
    const int blk = u >> 1;
    const int half = u & 1;
    const int group = blk < a.nb4 ? 0 : (blk < a.nb4 + a.nb6 ? 1 : 2);
    const FmtParams f = fmt_params(group);

    for (int r = 0; r < nrows; ++r) {
      const uint16_t* src = lds_rows + r * K;
      uint32_t h[16];
      uint32_t amax = 0;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        h[i] = src[p[i]];
        const uint32_t m = h[i] & 0x7FFFu;
        amax = m > amax ? m : amax;
      }
      // the other half of this block lives in the neighbouring lane
      const uint32_t other = (uint32_t)__shfl_xor((int)amax, 1);
      amax = other > amax ? other : amax;
      const int e = block_exponent(amax, f.emax);
      const int64_t row = row0 + r;

      if (group == 0) {
        uint32_t w0 = 0, w1 = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) w0 |= encode_bf16(h[i], e, f) << (4 * i);
#pragma unroll
        for (int i = 0; i < 8; ++i) w1 |= encode_bf16(h[8 + i], e, f) << (4 * i);
        uint8_t* dst = a.q4 + row * a.ld4 + (int64_t)blk * 16 + half * 8;
        *reinterpret_cast<uint2*>(dst) = make_uint2(w0, w1);
      } else if (group == 1) {
        // 16 six-bit codes = 96 bits: a little-endian bit stream
        uint32_t c[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) c[i] = encode_bf16(h[i], e, f);
        const uint32_t w0 = c[0] | (c[1] << 6) | (c[2] << 12) | (c[3] << 18) | (c[4] << 24) | (c[5] << 30);
        const uint32_t w1 =
            (c[5] >> 2) | (c[6] << 4) | (c[7] << 10) | (c[8] << 16) | (c[9] << 22) | (c[10] << 28);
        const uint32_t w2 = (c[10] >> 4) | (c[11] << 2) | (c[12] << 8) | (c[13] << 14) | (c[14] << 20) |
                            (c[15] << 26);
        uint8_t* dst = a.q6 + row * a.ld6 + (int64_t)(blk - a.nb4) * 24 + half * 12;
        uint32_t* d32 = reinterpret_cast<uint32_t*>(dst);
        d32[0] = w0;
        d32[1] = w1;
        d32[2] = w2;
        // An odd number of E3M2 blocks ends the row 8 bytes short of a 16-byte
        // boundary; those padding bytes are part of the layout and read as
        // zero codes by the GEMM's 16-byte loads.
        if (half == 1 && blk - a.nb4 == a.nb6 - 1 && (a.nb6 & 1)) {
          d32[3] = 0u;
          d32[4] = 0u;
        }
      } else {
        uint32_t w[4] = {0, 0, 0, 0};
#pragma unroll
        for (int i = 0; i < 16; ++i) w[i >> 2] |= encode_bf16(h[i], e, f) << (8 * (i & 3));
        uint8_t* dst = a.q8 + row * a.ld8 + (int64_t)(blk - a.nb4 - a.nb6) * 32 + half * 16;
        *reinterpret_cast<uint4*>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
      }
      if (half == 0) a.sc[row * a.ldsc + blk] = (uint8_t)(e + 127);
    }
  }
}

// Rows per workgroup: enough to amortise the sigma load, while keeping the
// LDS footprint near 32 KB so several workgroups stay resident per CU.
static int rows_per_block(int K) {
  int R = 16384 / K;
  return R < 1 ? 1 : (R > 4 ? 4 : R);
}

hipError_t launch_quantize(const QuantArgs& a, hipStream_t stream) {
  const int R = rows_per_block(a.K);
  const int units = a.K >> 4;
  int T = ((units + 63) / 64) * 64;
  if (T > 1024) T = 1024;
  const int64_t grid = (a.rows + R - 1) / R;
  const size_t lds = (size_t)R * a.K * sizeof(uint16_t);
  hipLaunchKernelGGL(quantize_rows_kernel, dim3((unsigned)grid), dim3(T), lds, stream, a, R);
  return hipGetLastError();
}

}  // namespace mm
