// Fused reorder-and-quantize (MicroMix Sec. 3.2 "Quantization kernel",
// Fig. "micromix-design" b): one pass over bf16 rows that gathers channels by
// sigma (Sec. 3.1), takes each 32-channel block's shared E8M0 scale and writes
// E2M1 / E3M2 / E4M3 codes for the three groups (Sec. 2.1 MX rule).
//
// HBM-bound design for gfx950, two kernels:
//  - the ring kernel (passes of two or more rows, K <= 8192; below the
//    pipelined one): producer wavefronts load each pass straight into an
//    LDS ring with global_load_lds_dwordx4, several passes in flight per CU,
//    and with the norm also sum each pass's squares one pass ahead;
//  - the pipelined kernel, as follows.
//  - a pass is `rpp` consecutive rows; the grid is sized to the number of
//    workgroups the chip holds at once, each XCD takes a contiguous range of
//    passes and its workgroups stride through it; one thread per (row,
//    32-channel block), so each thread always quantises the same block index
//    and keeps that block's 32 sigma entries in registers, as LDS byte
//    addresses, for the whole workgroup;
//  - rows arrive with 16-byte coalesced loads (the only HBM read) into
//    registers and are written to one of two LDS stages: the loads of pass
//    p+1 are in flight while pass p is quantised from the other stage;
//  - the gather is 32 LDS u16 reads per thread; the block absmax is a packed
//    16-bit max over the sign-cleared bf16 bits;
//  - the codes come from the gfx950 scaled conversions, which divide by the
//    E8M0 scale and round to nearest even (E2M1 and E4M3 two codes per
//    instruction, E3M2 one instruction per block giving the packed 24-byte bit
//    stream).  The E4M3 conversion does not saturate, so E4M3 inputs are first
//    clamped to 448 * scale, which is exact in bf16;
//  - consecutive lanes own consecutive blocks, so a wavefront's code stores
//    cover a contiguous span of each group.
//
// With the RMSNorm fused in front (the norm variant, App. D.2): the waves
// sum each staged row's squares in fp64 (a row split across several waves),
// every thread forms its row's factor r = fp32(1 / sqrt(mean(x^2) + eps)),
// and every gathered element becomes bf16(gamma * bf16(x * r)) (fp32
// products, round to nearest even) before the block absmax.  The weights in
// block order (gamma gathered by sigma) sit in LDS, four 16-byte pieces per
// block at (piece * nblk + block) * 16 so a wavefront's reads are
// conflict-free, in the unused tail of stage 0 when it has room; otherwise
// (one wide row per pass) each thread keeps its block's 32 weights in
// registers.
#include "kernels.hpp"

namespace mm {
namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x32 __attribute__((ext_vector_type(32)));
typedef short i16x2 __attribute__((ext_vector_type(2)));
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
typedef int i32x6 __attribute__((ext_vector_type(6)));
typedef uint32_t u32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// The second LDS stage sits at a fixed byte offset, so stage selection folds
// into the immediate offset of the LDS reads.  One stage holds at most this
// many bytes (rpp * K * 2).
constexpr int kStageOff = 32768;
constexpr int kMaxChunks = 4;  // 16-byte loads per thread per pass
constexpr int kMaxRowSlots = 256;  // row square sums of one pass (rows per pass, or waves, never exceed this)
// dynamic LDS at most: two stages, the dummy slot and the row square sums; or
// one 64 KB row, the dummy slot, 16 (row, part) sums and its 64 KB of weights
constexpr int kMaxLds = 2 * (2 * kStageOff) + 16 + 8 * 16;

typedef float f32x2 __attribute__((ext_vector_type(2)));

// LDS pointers built from 32-bit byte addresses (the base already added)
typedef const __attribute__((address_space(3))) uint16_t lds_u16_t;

__device__ __forceinline__ uint16_t lds_u16(uint32_t byte_addr) {
  return *reinterpret_cast<lds_u16_t*>((uintptr_t)byte_addr);
}

__device__ __forceinline__ uint32_t max_u16x2(uint32_t a, uint32_t b) {
  return __builtin_bit_cast(uint32_t,
                            __builtin_elementwise_max(__builtin_bit_cast(u16x2, a), __builtin_bit_cast(u16x2, b)));
}

__device__ __forceinline__ uint32_t min_u16x2(uint32_t a, uint32_t b) {
  return __builtin_bit_cast(uint32_t,
                            __builtin_elementwise_min(__builtin_bit_cast(u16x2, a), __builtin_bit_cast(u16x2, b)));
}

// Zero codes and scale byte for block j of step `step` of row n (padding).
template <int G>
__device__ __forceinline__ void zero_block(const QuantArgs& a, int64_t step, int64_t gstep, int64_t n, int j) {
  uint8_t* dst = a.q[G] + code_offset<G>(step, a.rp, n, j);
  if constexpr (G == 0) {
    *reinterpret_cast<uint4*>(dst) = make_uint4(0u, 0u, 0u, 0u);
  } else if constexpr (G == 1) {
    uint2* d = reinterpret_cast<uint2*>(dst);
    d[0] = d[1] = d[2] = make_uint2(0u, 0u);
  } else {
    *reinterpret_cast<uint4*>(dst) = make_uint4(0u, 0u, 0u, 0u);
    *reinterpret_cast<uint4*>(dst + 512) = make_uint4(0u, 0u, 0u, 0u);
  }
  a.sc[(gstep * a.rp + n) * kStepBlocks + j] = 0;
}

template <int G>
__device__ __forceinline__ void zero_tail(const QuantArgs& a, int64_t step, int64_t gstep, int64_t n, int j) {
  for (int jj = j + 1; jj < kStepBlocks; ++jj) zero_block<G>(a, step, gstep, n, jj);
}

// Quantise block b (local to its group) of row n from the LDS stage at byte
// offset `off` from the addresses; rows past a.rows are padding and quantise
// an all-zero block.  The thread that owns a group's last block also zeroes
// the padding blocks of that step.
template <bool kNorm>
__device__ __forceinline__ void quantize_block(const uint32_t (&addr)[32], uint32_t off, int group, bool last,
                                               const QuantArgs& a, int64_t n, int b, int gstep0,
                                               const uint32_t (&gpk)[16], float rn) {
  // gather: the block's 32 permuted channels, all reads issued before any
  // is used, then packed as 16 bf16 pairs
  uint16_t e[32];
#pragma unroll
  for (int i = 0; i < 32; ++i) e[i] = lds_u16(addr[i] + off);
  __builtin_amdgcn_sched_barrier(0);
  uint32_t d[16];
  const bool pad_row = n >= a.rows;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    u16x2 v;
    v.x = e[2 * i];
    v.y = e[2 * i + 1];
    d[i] = __builtin_bit_cast(uint32_t, v);
  }
  if constexpr (kNorm) {
    // bf16(gamma * bf16(x * r)): fp32 products, each rounded to nearest even;
    // four pairs at a time, so the temporaries of all sixteen are never live
    // together
#pragma unroll
    for (int i0 = 0; i0 < 16; i0 += 4) {
#pragma unroll
      for (int i = i0; i < i0 + 4; ++i) {
        const uint32_t w = d[i];
        const f32x2 t = {__uint_as_float(w << 16) * rn, __uint_as_float(w & 0xFFFF0000u) * rn};
        const uint32_t y = __builtin_bit_cast(uint32_t, __builtin_convertvector(t, bf16x2));
        const f32x2 u = {__uint_as_float(y << 16) * __uint_as_float(gpk[i] << 16),
                         __uint_as_float(y & 0xFFFF0000u) * __uint_as_float(gpk[i] & 0xFFFF0000u)};
        d[i] = __builtin_bit_cast(uint32_t, __builtin_convertvector(u, bf16x2));
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) d[i] = pad_row ? 0u : d[i];

  // absmax: bf16 magnitudes compare as unsigned integers
  uint32_t m[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) m[i] = d[i] & 0x7FFF7FFFu;
#pragma unroll
  for (int s = 8; s >= 1; s >>= 1)
#pragma unroll
    for (int i = 0; i < s; ++i) m[i] = max_u16x2(m[i], m[i + s]);
  const uint32_t amax = (m[0] & 0xFFFFu) > (m[0] >> 16) ? (m[0] & 0xFFFFu) : (m[0] >> 16);

  // Shared exponent e = floor(log2 amax) - emax, clamped below at -127: for
  // a bf16 amax with biased exponent E this is max(E - 127 - emax, -127); a
  // subnormal or zero amax (E = 0) lands on the clamp.  The E8M0 byte is e+127.
  const bool e2m3 = (a.fs & 1) != 0, e5m2 = (a.fs & 2) != 0;  // the alternative formats of groups 1 and 2
  const int emax = group == 0 ? 2 : (group == 1 ? (e2m3 ? 2 : 4) : (e5m2 ? 15 : 8));
  const int E = (int)(amax >> 7);
  const uint32_t sbyte = (uint32_t)(E - emax > 0 ? E - emax : 0);
  // the conversions read the scale's E8M0 exponent from an fp32 operand
  const float scale = __uint_as_float(sbyte << 23);

  const int64_t step = b >> 2;
  const int j = b & 3;
  const int64_t gstep = gstep0 + step;
  if (group == 0) {
    uint32_t w[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint32_t v = 0;
      v = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(v, __builtin_bit_cast(bf16x2, d[4 * q + 0]), scale, 0);
      v = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(v, __builtin_bit_cast(bf16x2, d[4 * q + 1]), scale, 1);
      v = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(v, __builtin_bit_cast(bf16x2, d[4 * q + 2]), scale, 2);
      v = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(v, __builtin_bit_cast(bf16x2, d[4 * q + 3]), scale, 3);
      w[q] = v;
    }
    *reinterpret_cast<uint4*>(a.q[0] + code_offset<0>(step, a.rp, n, j)) = make_uint4(w[0], w[1], w[2], w[3]);
    if (last) zero_tail<0>(a, step, gstep, n, j);
  } else if (group == 1) {
    u32x16 v;
    i32x6 c;
    if (e2m3) {
      // clamp the magnitudes to the largest E2M3 value, 7.5 * 2^e (exact in
      // bf16: biased exponent e + 129 = sbyte + 2, mantissa 0x70), keep the
      // signs; nothing then depends on how the conversion treats larger values
      const uint32_t lim = ((sbyte + 2u) << 7) | 0x70u;
      const uint32_t lim2 = lim | (lim << 16);
#pragma unroll
      for (int i = 0; i < 16; ++i) v[i] = min_u16x2(d[i] & 0x7FFF7FFFu, lim2) | (d[i] & 0x80008000u);
      c = __builtin_amdgcn_cvt_scalef32_pk32_fp6_bf16(__builtin_bit_cast(bf16x32, v), scale);
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i) v[i] = d[i];
      c = __builtin_amdgcn_cvt_scalef32_pk32_bf6_bf16(__builtin_bit_cast(bf16x32, v), scale);
    }
    uint2* dst = reinterpret_cast<uint2*>(a.q[1] + code_offset<1>(step, a.rp, n, j));
    dst[0] = make_uint2((uint32_t)c[0], (uint32_t)c[1]);
    dst[1] = make_uint2((uint32_t)c[2], (uint32_t)c[3]);
    dst[2] = make_uint2((uint32_t)c[4], (uint32_t)c[5]);
    if (last) zero_tail<1>(a, step, gstep, n, j);
  } else {
    // the largest finite value times 2^e in bf16, mantissa 0x60 (1.75): E4M3
    // 448 (biased exponent e + 127 + 8 = sbyte + 8), E5M2 57344 (sbyte + 15)
    const uint32_t lim = ((sbyte + (e5m2 ? 15u : 8u)) << 7) | 0x60u;
    const uint32_t lim2 = lim | (lim << 16);
    uint32_t w[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      // clamp the magnitudes, keep the signs
      const uint32_t c0 = min_u16x2(d[2 * q] & 0x7FFF7FFFu, lim2) | (d[2 * q] & 0x80008000u);
      const uint32_t c1 = min_u16x2(d[2 * q + 1] & 0x7FFF7FFFu, lim2) | (d[2 * q + 1] & 0x80008000u);
      i16x2 v = {0, 0};
      if (e5m2) {
        v = __builtin_amdgcn_cvt_scalef32_pk_bf8_bf16(v, __builtin_bit_cast(bf16x2, c0), scale, false);
        v = __builtin_amdgcn_cvt_scalef32_pk_bf8_bf16(v, __builtin_bit_cast(bf16x2, c1), scale, true);
      } else {
        v = __builtin_amdgcn_cvt_scalef32_pk_fp8_bf16(v, __builtin_bit_cast(bf16x2, c0), scale, false);
        v = __builtin_amdgcn_cvt_scalef32_pk_fp8_bf16(v, __builtin_bit_cast(bf16x2, c1), scale, true);
      }
      w[q] = __builtin_bit_cast(uint32_t, v);
    }
    uint8_t* dst = a.q[2] + code_offset<2>(step, a.rp, n, j);
    *reinterpret_cast<uint4*>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
    *reinterpret_cast<uint4*>(dst + 512) = make_uint4(w[4], w[5], w[6], w[7]);
    if (last) zero_tail<2>(a, step, gstep, n, j);
  }
  a.sc[(gstep * a.rp + n) * kStepBlocks + j] = (uint8_t)sbyte;
}

}  // namespace

// Launch shape: blockDim.x = roundup64(rpp * nblk) <= kMaxThreads threads;
// thread t owns pass-row t / nblk and block t % nblk; gridDim.x <= number of
// passes.  kPipe: two LDS stages of rpp * K * 2 <= kStageOff bytes, loads of
// the next pass overlap the current one; otherwise gridDim.x equals the
// number of passes and one stage holds up to 2 * kStageOff bytes.
// Sums of squares of the rpp rows staged at byte offset stage_off, spread
// over the workgroup's W waves: with rpp <= W each row gets W / rpp waves,
// each summing one contiguous part of it; otherwise each wave sums whole rows
// (rows strided by W).  Every (row, part) sum goes to slot
// row * row_parts(rpp, W) + part at sq_off; squares of bf16 values are exact
// in fp64, and the sums use four accumulators per lane and a fixed shuffle
// tree, so the result does not depend on timing.
__device__ __forceinline__ int row_parts(int rpp, int W) { return rpp <= W ? W / rpp : 1; }

__device__ __forceinline__ void row_square_sums(const u32x4* lds4, uint32_t stage_off, uint32_t sq_off, int rpp, int K) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, W = blockDim.x >> 6;
  const int chunks = K >> 3;
  const int parts = row_parts(rpp, W);
  const int first = rpp <= W ? wave / parts : wave;
  const int step = rpp <= W ? rpp : W;  // loop once when rows get several waves
  for (int pr = first; pr < rpp; pr += step) {
    const int part = rpp <= W ? wave % parts : 0;
    const int c0 = part * chunks / parts, c1 = (part + 1) * chunks / parts;
    const u32x4* row = lds4 + ((stage_off + (uint32_t)pr * K * 2) >> 4);
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    for (int c = c0 + lane; c < c1; c += 64) {
      const u32x4 v = row[c];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const double lo = (double)__uint_as_float(v[k] << 16), hi = (double)__uint_as_float(v[k] & 0xFFFF0000u);
        acc[k] += lo * lo;
        acc[k] += hi * hi;
      }
    }
    double s = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    if (lane == 0) reinterpret_cast<__attribute__((address_space(3))) double*>((uintptr_t)sq_off)[pr * parts + part] = s;
    if (rpp <= W) break;
  }
}

// fp32 row factor of pass-row pr from its part sums (after a barrier): the
// same operations, in the same order, in every thread of the row.
__device__ __forceinline__ float row_factor(uint32_t sq_off, int pr, int rpp, int K, float eps) {
  const int parts = row_parts(rpp, blockDim.x >> 6);
  const __attribute__((address_space(3))) double* sq =
      reinterpret_cast<const __attribute__((address_space(3))) double*>((uintptr_t)sq_off) + pr * parts;
  double s = sq[0];
  for (int k = 1; k < parts; ++k) s += sq[k];
  return (float)(1.0 / sqrt(s / (double)K + (double)eps));
}

// kNorm: 0 plain; 1 RMSNorm with the weights in registers; 2 RMSNorm with the
// block-order weights in LDS at byte offset gamma_off.
template <int kMaxThreads, bool kPipe, int kNorm>
__global__ __launch_bounds__(kMaxThreads) void quantize_rows_kernel(QuantArgs a, int rpp, int gamma_off) {
  extern __shared__ u32x4 lds4[];
  const int tid = threadIdx.x;
  const int T = blockDim.x;
  const int K = a.K;
  const int nblk = K >> 5;
  const int prow = tid / nblk;
  const int blk = tid - prow * nblk;
  const bool active = prow < rpp;
  const int stage_bytes = rpp * K * 2;
  const int nchunks = stage_bytes >> 4;  // 16-byte chunks per pass
  const int64_t passes = (a.rp + rpp - 1) / rpp;  // padding rows included

  // sigma of this thread's block as LDS byte addresses within a stage; an
  // out-of-range entry (a caller error) is clamped to stay inside the row
  uint32_t addr[32];
  const int base = (int)(uint32_t)(uintptr_t)lds4 + (active ? prow : 0) * K * 2;
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const int4 v = *reinterpret_cast<const int4*>(a.perm + (active ? blk : 0) * 32 + 4 * q);
    const int p[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) addr[4 * q + i] = (uint32_t)(base + 2 * ((unsigned)p[i] < (unsigned)K ? p[i] : 0));
  }
  // keep the full addresses in registers: otherwise the common base is
  // factored out and re-added before every LDS read
#pragma unroll
  for (int i = 0; i < 32; ++i) asm volatile("" : "+v"(addr[i]));
  // the norm weights of this thread's block, gathered by sigma, as bf16 pairs
  // (kNorm 2: written once to LDS by the threads of pass-row 0)
  uint32_t gpk[16];
  if constexpr (kNorm != 0) {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int4 v = *reinterpret_cast<const int4*>(a.perm + (active ? blk : 0) * 32 + 4 * q);
      const int p[4] = {v.x, v.y, v.z, v.w};
      uint32_t g[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) g[i] = a.gamma[(unsigned)p[i] < (unsigned)K ? p[i] : 0];
      gpk[2 * q] = g[0] | (g[1] << 16);
      gpk[2 * q + 1] = g[2] | (g[3] << 16);
    }
    if constexpr (kNorm == 2) {
      if (active && prow == 0)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          lds4[(gamma_off >> 4) + q * nblk + blk] = u32x4{gpk[4 * q], gpk[4 * q + 1], gpk[4 * q + 2], gpk[4 * q + 3]};
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) gpk[i] = 0u;
  }
  const int group = blk < a.nb[0] ? 0 : (blk < a.nb[0] + a.nb[1] ? 1 : 2);
  const int b = blk - (group >= 1 ? a.nb[0] : 0) - (group >= 2 ? a.nb[1] : 0);  // block within its group
  const int gstep0 = (group >= 1 ? a.steps[0] : 0) + (group >= 2 ? a.steps[1] : 0);
  const bool last = b == (group == 0 ? a.nb[0] : (group == 1 ? a.nb[1] : a.nb[2])) - 1;  // the group's last block

  // 16-byte chunk c of a pass lies in pass-row c / (K/8); rows past the end
  // are read from the last row (their results are never stored) and chunks
  // past the pass go to a 16-byte dummy slot after the stages, so every load
  // and LDS write is unconditional and in bounds
  const int chunks_per_row = K >> 3;
  const uint32_t dummy = (uint32_t)((kPipe ? kStageOff : 0) + stage_bytes);
  // row square sums of the pass being quantised (norm variant), after the dummy slot
  const uint32_t sq_off = (uint32_t)(uintptr_t)lds4 + dummy + 16;
  u32x4 buf[kMaxChunks];
#define MM_LOAD_PASS(P)                                                                              \
  {                                                                                                  \
    const int64_t r0_ = (int64_t)(P)*rpp;                                                            \
    _Pragma("unroll") for (int j = 0; j < kMaxChunks; ++j) {                                         \
      int c = tid + j * T;                                                                           \
      c = c < nchunks ? c : nchunks - 1;                                                             \
      const int r = c / chunks_per_row;                                                              \
      int64_t row = r0_ + r;                                                                         \
      row = row < a.rows ? row : a.rows - 1;                                                         \
      buf[j] = *reinterpret_cast<const u32x4*>(a.x + row * a.ldx + (int64_t)(c - r * chunks_per_row) * 8); \
    }                                                                                                \
  }
#define MM_STORE_PASS(STAGE)                                                                         \
  {                                                                                                  \
    _Pragma("unroll") for (int j = 0; j < kMaxChunks; ++j) {                                         \
      const int c = tid + j * T;                                                                     \
      const uint32_t off = c < nchunks ? (uint32_t)((STAGE)*kStageOff + c * 16) : dummy;            \
      lds4[off >> 4] = buf[j];                                                                       \
    }                                                                                                \
  }

  // Workgroups are dealt to the 8 XCDs round-robin; each XCD takes a
  // contiguous range of passes, so the rows of one 32-row group (which share
  // cache lines in the packed layout) are written through one XCD's L2.
  int64_t q, q_end, stride;
  if (gridDim.x % 8 == 0) {
    const int x = blockIdx.x & 7;
    q = passes * x / 8 + (blockIdx.x >> 3);
    q_end = passes * (x + 1) / 8;
    stride = gridDim.x / 8;
  } else {
    q = blockIdx.x;
    q_end = passes;
    stride = gridDim.x;
  }
  MM_LOAD_PASS(q);
  MM_STORE_PASS(0);
  __syncthreads();
  for (int i = 0; q < q_end; ++i, q += stride) {
    const bool more = kPipe && q + stride < q_end;
    if (more) MM_LOAD_PASS(q + stride);
    float rn = 0.0f;
    if constexpr (kNorm != 0) {
      row_square_sums(lds4, (uint32_t)((i & 1) * kStageOff), sq_off, rpp, K);
      __syncthreads();
      rn = row_factor(sq_off, active ? prow : 0, rpp, K, a.eps);
    }
    const int64_t row = q * rpp + prow;
    if (active && row < a.rp) {
      uint32_t gq[16];
      if constexpr (kNorm == 2) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const u32x4 v = lds4[(gamma_off >> 4) + k * nblk + blk];
          gq[4 * k] = v[0];
          gq[4 * k + 1] = v[1];
          gq[4 * k + 2] = v[2];
          gq[4 * k + 3] = v[3];
        }
      } else {
#pragma unroll
        for (int k = 0; k < 16; ++k) gq[k] = gpk[k];
      }
      if ((i & 1) == 0)
        quantize_block<kNorm != 0>(addr, 0u, group, last, a, row, b, gstep0, gq, rn);
      else
        quantize_block<kNorm != 0>(addr, (uint32_t)kStageOff, group, last, a, row, b, gstep0, gq, rn);
    }
    if (more) MM_STORE_PASS((i + 1) & 1);
    __syncthreads();
  }
#undef MM_LOAD_PASS
#undef MM_STORE_PASS
}

// ---------------------------------------------------------------------------
// Ring variant (K <= 8192): one workgroup per CU, persistent over
// a range of passes.  Four producer wavefronts move each pass's rows from HBM
// straight into an LDS slot with global_load_lds_dwordx4 (1 KB per wavefront
// instruction, no register staging); a ring of kRingSlots slots keeps up to
// kRingSlots - 1 passes, about 96 KB per CU, in flight, where the pipelined
// kernel above has at most one pass of register-staged loads per workgroup.
// Eight consumer wavefronts quantise exactly as above (thread t owns
// pass-row t / nblk and block t % nblk).  One s_barrier per pass hands a
// landed slot to the consumers and the slot they have finished back to the
// producers.  Only the producers load and only the consumers store, so each
// producer's vmcnt counts its own loads alone and the wait for a pass is one
// constant: every producer issues NPER loads for every pass (loads past the
// pass's bytes repeat its last one, into the same LDS bytes).
// ---------------------------------------------------------------------------
constexpr int kRingSlots = 4;
constexpr int kRingSlotMax = 32768;  // bytes of one pass's rows at most (a slot adds up to 1 KB of padding)
constexpr int kProducerWaves = 4;
constexpr int kConsumerWaves = 8;
constexpr int kRingThreads = 64 * (kProducerWaves + kConsumerWaves);
constexpr int kMaxRingRows = 64 * kConsumerWaves;  // rows per pass at most (one block per row)

// vmcnt-only wait (expcnt and lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Workgroup barrier without the wait for loads in flight that __syncthreads
// adds (the producers' loads must stay in flight across it).
__device__ __forceinline__ void bare_barrier() { asm volatile("s_barrier" ::: "memory"); }

__device__ __forceinline__ uint32_t uni32(uint32_t v) { return (uint32_t)__builtin_amdgcn_readfirstlane((int)v); }
__device__ __forceinline__ const uint8_t* uni_ptr(const uint8_t* p) {
  const uint64_t v = (uint64_t)p;
  const uint64_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
  const uint64_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(v >> 32));
  return (const uint8_t*)(lo | (hi << 32));
}

// Direct global -> LDS load: lane i's 16 bytes at sbase + voff land at M0 +
// 16 i.  Inline asm, so the compiler neither tracks nor waits for it; the
// producers' explicit vmcnt waits do.  The s_nop covers the M0 write.  The
// rows are read once, so the load is marked non-temporal (nt): their lines
// go first when the L2 evicts, and the partly written lines of the packed
// codes (runs of a few rows that other workgroups complete) stay there to be
// merged (8192 x 5120: 31.6 -> 28.6 us).
__device__ __forceinline__ void dma16(uint32_t voff, const uint8_t* sbase, uint32_t lds) {
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 nt" : : "v"(voff), "s"(sbase), "{m0}"(lds) : "memory");
}

// Square sums of the rows of the pass in the slot at `slot` (row r at r *
// row_stride), one row per producer wavefront at a time, into the fp64
// words at `sums`: four accumulators per lane over 16-byte reads, then a
// fixed shuffle tree, so the result does not depend on timing (squares of
// bf16 values are exact in fp64).
__device__ __forceinline__ void ring_row_sums(uint32_t slot, int row_stride, int rpp, int K, int pw, int lane,
                                              uint32_t sums) {
  for (int r = pw; r < rpp; r += kProducerWaves) {
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    for (int c = lane; c < (K >> 3); c += 64) {
      const u32x4 v = *reinterpret_cast<const __attribute__((address_space(3))) u32x4*>(
          (uintptr_t)(slot + (uint32_t)r * (uint32_t)row_stride + (uint32_t)c * 16u));
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const double lo = (double)__uint_as_float(v[k] << 16), hi = (double)__uint_as_float(v[k] & 0xFFFF0000u);
        acc[k] += lo * lo;
        acc[k] += hi * hi;
      }
    }
    double t = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    for (int o = 32; o > 0; o >>= 1) t += __shfl_xor(t, o);
    if (lane == 0) *reinterpret_cast<__attribute__((address_space(3))) double*>((uintptr_t)(sums + 8u * r)) = t;
  }
}

// kNorm: the RMSNorm in front.  The producers then also sum each pass's
// squares one pass ahead (after the barrier at which pass k + 1 has landed,
// into one of two sum buffers), so the consumers of pass k find its row
// factors ready; this keeps one pass fewer in flight.
template <int NPER, bool kNorm>
__global__ __launch_bounds__(kRingThreads, 1) void quantize_ring_kernel(QuantArgs a, int rpp, int row_stride,
                                                                       int slot_stride) {
  extern __shared__ __attribute__((aligned(1024))) uint8_t ring[];
  const uint32_t lds0 = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint8_t*)ring;
  // the norm's row square sums: two buffers of kMaxRingRows fp64 words after the slots
  const uint32_t sums0 = lds0 + (uint32_t)kRingSlots * (uint32_t)slot_stride;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int K = a.K;
  const int nblk = K >> 5;
  const int64_t passes = (a.rp + rpp - 1) / rpp;  // padding rows included

  // this workgroup's passes: each XCD a contiguous range (the rows of a
  // 32-row group share cache lines in the packed layout), its workgroups
  // strided through it
  int64_t q, q_end, stride;
  if (gridDim.x % 8 == 0) {
    const int x = blockIdx.x & 7;
    q = passes * x / 8 + (blockIdx.x >> 3);
    q_end = passes * (x + 1) / 8;
    stride = gridDim.x / 8;
  } else {
    q = blockIdx.x;
    q_end = passes;
    stride = gridDim.x;
  }
  if (q >= q_end) return;  // uniform over the workgroup
  const int64_t nk = (q_end - q + stride - 1) / stride;

  if (wave >= kConsumerWaves) {
    // producer: pass k goes to slot k % kRingSlots, row r of the pass at
    // r * row_stride in the slot; wavefront pw issues the pass's 1 KB pieces
    // pw, pw + 4, ... (a piece past the last repeats the last); passes past
    // the workgroup's last repeat it
    const int pw = wave - kConsumerWaves;
    const int lane = tid & 63;
    const int cpr = K >> 3;  // 16-byte chunks per row
    // padded rows (row_stride > 2K, K a multiple of 512): whole 1 KB pieces
    // per row; otherwise rows back to back, pieces across row ends
    const bool padded = row_stride != 2 * K;
    const int ipr = cpr >> 6;  // pieces per row when padded
    const int nchunks = rpp * cpr;
    const int ninstr = padded ? rpp * ipr : (nchunks + 63) >> 6;
    auto issue = [&](int64_t k) {
      const int64_t kk = k < nk ? k : nk - 1;
      const int64_t r0 = (q + kk * stride) * rpp;
      // rows past the input are read from its last row (their blocks
      // quantise as padding and never use them)
      const int64_t rb = r0 < a.rows ? r0 : a.rows - 1;
      const uint8_t* base = uni_ptr(reinterpret_cast<const uint8_t*>(a.x + rb * a.ldx));
      const uint32_t slot = lds0 + (uint32_t)(k % kRingSlots) * (uint32_t)slot_stride;
#pragma unroll
      for (int j = 0; j < NPER; ++j) {
        int i = pw + kProducerWaves * j;
        i = i < ninstr ? i : ninstr - 1;
        int rr, c;  // row within the pass, chunk within the row
        uint32_t dst;
        if (padded) {
          rr = i / ipr;
          const int ii = i - rr * ipr;
          c = ii * 64 + lane;
          dst = slot + (uint32_t)rr * (uint32_t)row_stride + (uint32_t)ii * 1024u;
        } else {
          int cc = i * 64 + lane;
          cc = cc < nchunks ? cc : nchunks - 1;
          rr = cc / cpr;
          c = cc - rr * cpr;
          dst = slot + (uint32_t)i * 1024u;
        }
        int64_t row = r0 + rr;
        row = row < a.rows ? row : a.rows - 1;
        const uint32_t voff = (uint32_t)((row - rb) * a.ldx * 2 + (int64_t)c * 16);
        dma16(voff, base, uni32(dst));
      }
    };
    for (int k = 0; k < kRingSlots - 1; ++k) issue(k);
    if constexpr (kNorm) {
      // the sums of pass 0 before the consumers start
      wait_vmcnt<(kRingSlots - 2) * NPER>();
      bare_barrier();
      ring_row_sums(lds0, row_stride, rpp, K, pw, lane, sums0);
    }
    for (int64_t k = 0; k < nk; ++k) {
      // pass k landed (this wavefront's loads; the kRingSlots - 2 passes
      // after it may still be in flight), then everyone's; with the norm
      // pass k + 1 too, whose sums follow
      wait_vmcnt<(kRingSlots - (kNorm ? 3 : 2)) * NPER>();
      bare_barrier();
      // the consumers are done with pass k - 1: refill its slot
      issue(k + kRingSlots - 1);
      if constexpr (kNorm)
        if (k + 1 < nk)
          ring_row_sums(lds0 + (uint32_t)((k + 1) % kRingSlots) * (uint32_t)slot_stride, row_stride, rpp, K, pw,
                        lane, sums0 + (uint32_t)((k + 1) & 1) * 8u * kMaxRingRows);
    }
    wait_vmcnt<0>();  // no load may land after the workgroup's LDS is released
    return;
  }

  // consumer: thread t owns block t / rpp of pass-row t % rpp, so the
  // lanes that store one block's codes hold consecutive rows, whose codes
  // are consecutive in the packed layout (one contiguous run per block
  // instead of one 16-byte piece per lane); with padded rows those lanes'
  // gather reads fall on different banks
  const int blk = tid / rpp;
  const int prow = tid - blk * rpp;
  const bool active = blk < nblk;
  uint32_t addr[32];
  const uint32_t base = lds0 + (uint32_t)prow * (uint32_t)row_stride;
#pragma unroll
  for (int qq = 0; qq < 8; ++qq) {
    const int4 v = *reinterpret_cast<const int4*>(a.perm + (active ? blk : 0) * 32 + 4 * qq);
    const int p[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) addr[4 * qq + i] = base + 2u * (uint32_t)((unsigned)p[i] < (unsigned)K ? p[i] : 0);
  }
#pragma unroll
  for (int i = 0; i < 32; ++i) asm volatile("" : "+v"(addr[i]));
  // the norm weights of this thread's block, gathered by sigma, as bf16 pairs
  uint32_t gpk[16];
  if constexpr (kNorm) {
#pragma unroll
    for (int qq = 0; qq < 8; ++qq) {
      const int4 v = *reinterpret_cast<const int4*>(a.perm + (active ? blk : 0) * 32 + 4 * qq);
      const int p[4] = {v.x, v.y, v.z, v.w};
      uint32_t gg[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) gg[i] = a.gamma[(unsigned)p[i] < (unsigned)K ? p[i] : 0];
      gpk[2 * qq] = gg[0] | (gg[1] << 16);
      gpk[2 * qq + 1] = gg[2] | (gg[3] << 16);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) gpk[i] = 0u;
  }
  const int bb = active ? blk : 0;
  const int group = bb < a.nb[0] ? 0 : (bb < a.nb[0] + a.nb[1] ? 1 : 2);
  const int b = bb - (group >= 1 ? a.nb[0] : 0) - (group >= 2 ? a.nb[1] : 0);
  const int gstep0 = (group >= 1 ? a.steps[0] : 0) + (group >= 2 ? a.steps[1] : 0);
  const bool last = b == (group == 0 ? a.nb[0] : (group == 1 ? a.nb[1] : a.nb[2])) - 1;
  if constexpr (kNorm) bare_barrier();  // the producers' barrier before pass 0's sums
  for (int64_t k = 0; k < nk; ++k) {
    bare_barrier();
    const int64_t row = (q + k * stride) * rpp + prow;
    float rn = 0.0f;
    if constexpr (kNorm) {
      // fp32(1 / sqrt(mean(x^2) + eps)) from the row's fp64 square sum
      const double sq = *reinterpret_cast<const __attribute__((address_space(3))) double*>(
          (uintptr_t)(sums0 + (uint32_t)(k & 1) * 8u * kMaxRingRows + 8u * (uint32_t)prow));
      rn = (float)(1.0 / sqrt(sq / (double)K + (double)a.eps));
    }
    if (active && row < a.rp)
      quantize_block<kNorm>(addr, (uint32_t)(k % kRingSlots) * (uint32_t)slot_stride, group, last, a, row, b,
                            gstep0, gpk, rn);
    // every read of this slot is done before the barrier that frees it
    __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (3 << 14));
  }
}

// Allow more than 64 KB of dynamic LDS (two 32 KB stages plus the dummy
// slot and the row square sums, or one wide row and its weights).
template <int kMaxThreads, bool kPipe, int kNorm>
static hipError_t allow_lds(size_t bytes) {
  static bool done = false;
  if (done || bytes <= 65536) return hipSuccess;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(quantize_rows_kernel<kMaxThreads, kPipe, kNorm>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, kMaxLds);
  if (e == hipSuccess) done = true;
  return e;
}

// Workgroups of the pipelined kernel resident on the current device at once
// (per-CU occupancy times CU count), cached per thread for the last shape.
template <int kNorm>
static hipError_t resident_workgroups(int T, size_t lds, int* cap) {
  thread_local int last_dev = -1, last_T = 0, last_cap = 0;
  thread_local size_t last_lds = 0;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev != last_dev || T != last_T || lds != last_lds) {
    int per_cu = 0, cus = 0;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, quantize_rows_kernel<512, true, kNorm>, T, lds);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    last_dev = dev;
    last_T = T;
    last_lds = lds;
    last_cap = (per_cu < 1 ? 1 : per_cu) * (cus < 1 ? 1 : cus);
  }
  *cap = last_cap;
  return hipSuccess;
}

template <int kNorm>
static hipError_t launch_pipelined(const QuantArgs& a, int rpp, int T, size_t lds, int gamma_off, hipStream_t stream) {
  hipError_t e = allow_lds<512, true, kNorm>(lds);
  if (e != hipSuccess) return e;
  // one wave of workgroups: as many as the chip holds at once
  int cap = 0;
  e = resident_workgroups<kNorm>(T, lds, &cap);
  if (e != hipSuccess) return e;
  const int64_t passes = (a.rp + rpp - 1) / rpp;
  const int64_t grid = passes < cap ? passes : cap;
  hipLaunchKernelGGL((quantize_rows_kernel<512, true, kNorm>), dim3((unsigned)grid), dim3(T), lds, stream, a, rpp,
                     gamma_off);
  return hipGetLastError();
}

// CUs of the current device (cached per thread for the last device).
static hipError_t device_cus(int* cus) {
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

template <int NPER, bool kNorm>
static hipError_t launch_ring_n(const QuantArgs& a, int rpp, int row_stride, int slot_stride, int grid,
                                hipStream_t stream) {
  static bool attr = false;
  constexpr size_t kSumBytes = 2 * 8 * kMaxRingRows;
  const size_t lds = (size_t)kRingSlots * slot_stride + (kNorm ? kSumBytes : 0);
  if (!attr) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(quantize_ring_kernel<NPER, kNorm>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       kRingSlots * (kRingSlotMax + 1024) + kSumBytes);
    if (e != hipSuccess) return e;
    attr = true;
  }
  hipLaunchKernelGGL((quantize_ring_kernel<NPER, kNorm>), dim3((unsigned)grid), dim3(kRingThreads), lds, stream, a,
                     rpp, row_stride, slot_stride);
  return hipGetLastError();
}

template <bool kNorm>
static hipError_t launch_ring_norm(const QuantArgs& a, int nper, int rpp, int row_stride, int slot_stride, int grid,
                                   hipStream_t stream) {
  if (nper <= 1) return launch_ring_n<1, kNorm>(a, rpp, row_stride, slot_stride, grid, stream);
  if (nper <= 2) return launch_ring_n<2, kNorm>(a, rpp, row_stride, slot_stride, grid, stream);
  if (nper <= 4) return launch_ring_n<4, kNorm>(a, rpp, row_stride, slot_stride, grid, stream);
  return launch_ring_n<8, kNorm>(a, rpp, row_stride, slot_stride, grid, stream);
}

// The ring kernel for K <= 8192 (passes of two or more rows), with or
// without the norm; *used = false leaves the launch to the kernels below.
static hipError_t launch_ring(const QuantArgs& a, hipStream_t stream, bool* used) {
  *used = false;
  const int K = a.K;
  const int nblk = K >> 5;
  if (nblk > 64 * kConsumerWaves || 2 * K > kRingSlotMax) return hipSuccess;
  // rows per pass: as many as the consumer threads and one slot take
  int rpp = 64 * kConsumerWaves / nblk;
  if (rpp * 2 * K > kRingSlotMax) rpp = kRingSlotMax / (2 * K);
  int cus = 0;
  hipError_t e = device_cus(&cus);
  if (e != hipSuccess) return e;
  // few rows (under eight passes per workgroup), plain quantiser: halve the
  // pass while it keeps two or more rows, so that each workgroup's ring has
  // more passes to overlap (2048 x 4096: 9.6 -> 8.8 us; 4096 x 4096, with
  // the streamed loads: 15.5 -> 14.1 us; with the norm the producers' row
  // sums then lose half their wavefronts, so not there)
  while (a.norm == 0 && rpp >= 4 && (a.rp + rpp - 1) / rpp < 8 * (int64_t)cus) rpp /= 2;
  // one row per pass (K > 8192): the pipelined kernel measured faster
  // there (K = 14336: 35 us against 42 us for 4096 rows)
  if (rpp < 2) return hipSuccess;
  // per-lane load offsets are 32-bit, relative to the pass's first row
  if ((int64_t)rpp * a.ldx * 2 + (int64_t)K * 2 >= ((int64_t)1 << 32)) return hipSuccess;
  // rows padded by 16 bytes in LDS when they are whole 1 KB loads (K a
  // multiple of 512) and the pass has several, so the gather reads of one
  // block's rows fall on different banks
  const bool padded = K % 512 == 0 && rpp > 1;
  const int row_stride = padded ? 2 * K + 16 : 2 * K;
  const int bytes = rpp * row_stride;
  const int slot_stride = (bytes + 1023) / 1024 * 1024;  // the last 1 KB load may run past the pass's bytes
  const int ninstr = padded ? rpp * (2 * K / 1024) : (bytes + 1023) / 1024;
  const int nper = (ninstr + kProducerWaves - 1) / kProducerWaves;
  const int64_t passes = (a.rp + rpp - 1) / rpp;
  const int grid = (int)(passes < cus ? passes : cus);
  *used = true;
  if (a.norm != 0) return launch_ring_norm<true>(a, nper, rpp, row_stride, slot_stride, grid, stream);
  return launch_ring_norm<false>(a, nper, rpp, row_stride, slot_stride, grid, stream);
}

static hipError_t launch_quantize_rows(const QuantArgs& a, hipStream_t stream) {
  const int K = a.K;
  const int nblk = K >> 5;
  const bool norm = a.norm != 0;
  bool ring_used = false;
  hipError_t re = launch_ring(a, stream, &ring_used);
  if (re != hipSuccess || ring_used) return re;
  // A row wider than one stage (K > 16384) is quantised without overlap, one
  // row per workgroup of K/32 threads (up to 1024); with the norm its weights
  // follow the row, the dummy slot and the (row, part) sums in LDS.
  if (K * 2 > kStageOff) {
    const int T = (nblk + 63) / 64 * 64;
    const int gamma_off = K * 2 + 16 + 8 * 16;
    if (norm) {
      const size_t lds = (size_t)gamma_off + (size_t)K * 2;
      hipError_t e = allow_lds<1024, false, 2>(lds);
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL((quantize_rows_kernel<1024, false, 2>), dim3((unsigned)a.rp), dim3(T), lds, stream, a, 1,
                         gamma_off);
    } else {
      const size_t lds = (size_t)K * 2 + 16;
      hipError_t e = allow_lds<1024, false, 0>(lds);
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL((quantize_rows_kernel<1024, false, 0>), dim3((unsigned)a.rp), dim3(T), lds, stream, a, 1, 0);
    }
    return hipGetLastError();
  }
  // rows per pass: the fewest idle lanes (ties: more rows) among launches of
  // up to 512 threads, stopping at the first of at least 256 threads; a pass
  // must fit one LDS stage
  const int max_rpp = kStageOff / (K * 2);
  int rpp = 1;
  double best = 2.0;
  for (int r = 1; r <= max_rpp && r * nblk <= 512; ++r) {
    const int t = (r * nblk + 63) / 64 * 64;
    const double idle = (double)(t - r * nblk) / t;
    if (idle <= best) {
      best = idle;
      rpp = r;
    }
    if (t >= 256) break;
  }
  if (rpp > kMaxRowSlots) return hipErrorInvalidValue;  // cannot happen: rpp * nblk <= 512
  const int T = (rpp * nblk + 63) / 64 * 64;
  // two stages plus the 16-byte dummy slot (and the (row, part) square sums)
  size_t lds = (size_t)kStageOff + (size_t)rpp * K * 2 + 16;
  if (!norm) return launch_pipelined<0>(a, rpp, T, lds, 0, stream);
  const int slots = rpp > T / 64 ? rpp : T / 64;  // max(rpp, waves)
  lds += (size_t)slots * 8;
  // the block-order weights fit the unused tail of stage 0
  if ((rpp + 1) * K * 2 <= kStageOff) return launch_pipelined<2>(a, rpp, T, lds, rpp * K * 2, stream);
  return launch_pipelined<1>(a, rpp, T, lds, 0, stream);
}

hipError_t launch_quantize(const QuantArgs& a, hipStream_t stream) {
  if (a.rows == 0) return hipSuccess;
  return launch_quantize_rows(a, stream);
}

}  // namespace mm
