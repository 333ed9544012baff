// Shared pieces of the MicroMix mixed-precision GEMM kernels (gfx950).
//
// The product Y = A W^T of Sec. 2.1 eq. 1 is computed by the CDNA4
// block-scaled MFMA V_MFMA_SCALE_F32_16X16X128_F8F6F4, which multiplies two
// 16 x 128 operand tiles whose 32-element blocks each carry an E8M0 scale, and
// accumulates in fp32.  All three groups (E2M1, E3M2, E4M3) feed the same
// accumulator (Sec. 3.2 "GEMM kernel"); the format is an instruction
// immediate, so each group runs its own specialised K loop.
//
// Register layout of one 16 x 128 operand tile in a wavefront (lane = 16 g + r,
// r = tile row, g = 0..3), as measured on gfx950:
//   E2M1 / E3M2: the lane holds the 32 elements of block g (K 32g .. 32g+31),
//                packed densely (4 or 6 bits per element, little-endian) in
//                the first 4 or 6 registers;
//   E4M3:        the lane holds K 16g .. 16g+15 in bytes 0-15 and
//                K 64+16g .. 64+16g+15 in bytes 16-31;
//   scale:       the E8M0 byte for (row r, block b) comes from lane 16 b + r
//                (byte 0 of the scale register with op_sel 0), for every format.
// The fp32 result tile: lane 16 g + r, register q holds C[4 g + q][r], where
// C's row indexes the first operand and its column the second.
#pragma once

#include "kernels.hpp"
#include "mx_device.hpp"

namespace mm {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// kStream: a non-temporal load (data read once: its L2 lines go first).
template <bool kStream = false>
__device__ __forceinline__ uint4 gload16(const void* p) {
  const __attribute__((address_space(1))) u32x4* q = (const __attribute__((address_space(1))) u32x4*)(p);
  u32x4 v;
  if constexpr (kStream) v = __builtin_nontemporal_load(q);
  else v = *q;
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint2 gload8(const void* p) {
  const u32x2 v = *(const __attribute__((address_space(1))) u32x2*)(p);
  return make_uint2(v.x, v.y);
}

// MFMA format selector of a group.
// MFMA format selector of a group under format set fs (bit 0: the 6-bit
// group is E2M3 instead of E3M2; bit 1: the 8-bit group is E5M2 instead of
// E4M3).
__host__ __device__ constexpr int group_fmt(int group, int fs) {
  return group == 0 ? kE2M1 : (group == 1 ? ((fs & 1) ? kE2M3 : kE3M2) : ((fs & 2) ? kE5M2 : kE4M3));
}

// One lane's 16 x 128 operand fragment (16 x 16 x 128 form, lane 16 g + r)
// straight from the packed layout: row n, step `step` of group G.  The padded
// layout makes every step whole, so there is no bounds logic here.  kStream
// makes the E2M1 and E4M3 loads non-temporal; the E3M2 ones stay plain (a
// lane's 24 bytes come in two loads whose cache lines other lanes share, and
// streamed lines can be gone before the second load).
template <int G, bool kStream = false>
__device__ __forceinline__ v8i load_frag16_global(const uint8_t* base, int64_t rp, int64_t n, int64_t step, int g) {
  v8i v;
  if constexpr (G == 0) {
    const uint4 d = gload16<kStream>(base + code_offset<0>(step, rp, n, g));
    v[0] = (int)d.x;
    v[1] = (int)d.y;
    v[2] = (int)d.z;
    v[3] = (int)d.w;
    v[4] = v[5] = v[6] = v[7] = 0;
  } else if constexpr (G == 1) {
    const uint8_t* s = base + code_offset<1>(step, rp, n, g);
    const uint2 d0 = gload8(s), d1 = gload8(s + 8), d2 = gload8(s + 16);
    v[0] = (int)d0.x;
    v[1] = (int)d0.y;
    v[2] = (int)d1.x;
    v[3] = (int)d1.y;
    v[4] = (int)d2.x;
    v[5] = (int)d2.y;
    v[6] = v[7] = 0;
  } else {
    // channels 16g .. 16g+15: block g/2, half g%2, i.e. record slot g; and
    // channels 64+16g ..: block 2 + g/2, half g%2, record slot 4 + g
    const uint8_t* s = base + code_offset<2>(step, rp, n, 0);
    const uint4 lo = gload16<kStream>(s + g * 512);
    const uint4 hi = gload16<kStream>(s + (4 + g) * 512);
    v[0] = (int)lo.x;
    v[1] = (int)lo.y;
    v[2] = (int)lo.z;
    v[3] = (int)lo.w;
    v[4] = (int)hi.x;
    v[5] = (int)hi.y;
    v[6] = (int)hi.z;
    v[7] = (int)hi.w;
  }
  return v;
}

// E8M0 scale of block j of global step t of row n.
__device__ __forceinline__ int load_scale(const uint8_t* sc, int64_t rp, int64_t t, int64_t n, int j) {
  return *(const __attribute__((address_space(1))) uint8_t*)(sc + (t * rp + n) * kStepBlocks + j);
}

// acc = acc + A(group G) x B(group G) with per-block E8M0 scales sa / sb.
// The format selectors must reach the builtin as integer constants (they are
// instruction immediates), hence the constexpr locals.
#define MM_MFMA_GROUP(G, FS, acc, a, b, sa, sb)                                                     \
  do {                                                                                              \
    constexpr int mm_fmt_ = group_fmt(G, FS);                                                       \
    (acc) = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4((a), (b), (acc), mm_fmt_, mm_fmt_, 0, \
                                                             (sa), 0, (sb));                        \
  } while (0)

typedef float v16f __attribute__((ext_vector_type(16)));

// The 32 x 32 x 64 form (V_MFMA_SCALE_F32_32X32X64_F8F6F4): lane 32 g + r
// holds row r; E2M1 / E3M2 lanes hold block g of the 64-channel step, E4M3
// lanes hold channels 16g .. 16g+15 and 32+16g .. 32+16g+15; the scale of
// (row r, block b) comes from lane 32 b + r.  Result: lane 32 g + r,
// register q holds C[8 (q/4) + 4 g + q%4][r].  On gfx950 this form runs E2M1
// and E3M2 well above the 16 x 16 x 128 form's rate.
#define MM_MFMA32_GROUP(G, FS, acc, a, b, sa, sb)                                                   \
  do {                                                                                              \
    constexpr int mm_fmt_ = group_fmt(G, FS);                                                       \
    (acc) = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4((a), (b), (acc), mm_fmt_, mm_fmt_, 0,  \
                                                            (sa), 0, (sb));                         \
  } while (0)

// fp32 -> bf16, round to nearest even (finite inputs; overflow gives inf).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// Two fp32 values rounded to nearest even as a packed bf16 pair (a in the low
// half): one gfx950 conversion instruction (v_cvt_pk_bf16_f32) instead of
// the integer sequence above per value.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2_rne(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}

// Store lane's 4 consecutive output columns n..n+3 of row m.
__device__ __forceinline__ void store_out4(const GemmArgs& a, int64_t m, int64_t n, const v4f& c, int64_t M,
                                           int64_t N) {
  if (m >= M) return;
  uint16_t* dst = a.y + m * a.ldy + n;
  if (n + 3 < N) {
    const uint32_t lo = pack_bf16x2_rne(c[0], c[1]);
    const uint32_t hi = pack_bf16x2_rne(c[2], c[3]);
    *reinterpret_cast<uint2*>(dst) = make_uint2(lo, hi);
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (n + q < N) dst[q] = (uint16_t)f32_to_bf16_rne(c[q]);
  }
}

}  // namespace mm
