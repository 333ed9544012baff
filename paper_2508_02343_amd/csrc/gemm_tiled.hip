// Mixed MX GEMM for prefill shapes (many activation rows): compute-bound on
// the block-scaled MFMA, so operand tiles are staged in LDS and reused by
// the whole workgroup.
//
// Workgroup tile: BN weight rows (output columns n) x BM activation rows
// (output rows m), four wavefronts in a 2 x 2 grid, each owning a
// (BN/2) x (BM/2) block of 16 x 16 fp32 MFMA accumulators.  The K loop visits
// the E2M1 group, then E3M2, then E4M3 (Sec. 3.1 group order), 128 channels
// (4 MX blocks) per step, all accumulating into the same registers
// (Sec. 3.2 "GEMM kernel": one fp32 accumulation, one bf16 rounding).
//
// Memory pipeline (gfx950): operand bytes and their E8M0 scales go straight
// from global memory into LDS with global_load_lds_dwordx4 / _dword, through
// a ring of as many stages as 160 KB of LDS holds for the group's format
// (E2M1 rows are 64 bytes per step, E3M2 96, E4M3 128), so several steps are
// in flight while the MFMAs work on the oldest one.  Completion is tracked
// with explicit vmcnt waits and bare s_barrier (a __syncthreads fence would
// wait for every load in flight).  Rows are stored with a per-format chunk
// swizzle so that a wavefront's fragment reads spread over the LDS banks.
// Workgroups are mapped to tiles XCD by XCD and in groups of weight tiles,
// so the tiles that run together on one XCD share its L2.
#include "gemm_common.hpp"

namespace mm {

namespace tiled {

constexpr int kThreads = 256;
constexpr int kLdsBytes = 160 * 1024;
constexpr int kRingBytes = kLdsBytes - 16;  // the last 16 bytes hold constants
constexpr int kOneOffset = kRingBytes;      // LDS byte holding E8M0 127 (1.0)

__host__ __device__ constexpr int row_bytes(int G) { return G == 0 ? 64 : (G == 1 ? 96 : 128); }
__host__ __device__ constexpr int chunks(int G) { return row_bytes(G) / 16; }

template <int G, int BN, int BM>
struct Plan {
  static constexpr int kRows = BN + BM;
  static constexpr int kCodeBytes = kRows * row_bytes(G);     // codes of one stage
  static constexpr int kStageBytes = kCodeBytes + kRows * 8;  // + 2 scale words per row
  static constexpr int kStages = kRingBytes / kStageBytes;
  static constexpr int kCodeLoads = kRows * chunks(G) / kThreads;  // dwordx4 DMA per thread
  static constexpr int kScaleLoads = kRows * 2 / kThreads;         // dword DMA per thread
  static constexpr int kLoads = kCodeLoads + kScaleLoads;
  static_assert(kStages >= 2, "LDS ring needs two stages");
  static_assert(kRows * chunks(G) % kThreads == 0 && kRows * 2 % kThreads == 0, "tile / thread mismatch");
  static_assert((kStages - 2) * kLoads < 64, "vmcnt range");
};

// Physical 16-byte chunk of logical chunk c in row r (and its inverse).
// E2M1 / E4M3 rows use an XOR swizzle; E3M2 blocks (24 bytes) straddle
// chunks, so its rows are rotated by one chunk instead.
template <int G>
__device__ __forceinline__ int swz(int c, int r) {
  if constexpr (G == 0) return c ^ ((r >> 1) & 3);
  else if constexpr (G == 1) return ((r >> 2) & 1) ? (c == 5 ? 0 : c + 1) : c;
  else return c ^ (r & 7);
}
template <int G>
__device__ __forceinline__ int unswz(int c, int r) {
  if constexpr (G == 1) return ((r >> 2) & 1) ? (c == 0 ? 5 : c - 1) : c;
  else return swz<G>(c, r);
}

// vmcnt-only wait (expcnt and lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// lgkmcnt(0) only.
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (3 << 14)); }

// Workgroup barrier that is also a compiler memory barrier but, unlike
// __syncthreads, adds no wait for loads in flight.
__device__ __forceinline__ void barrier() { asm volatile("s_barrier" ::: "memory"); }

// 32-bit LDS address of a pointer into dynamic shared memory.
__device__ __forceinline__ uint32_t lds_addr(const uint8_t* p) {
  return (uint32_t)(size_t)(const __attribute__((address_space(3))) uint8_t*)p;
}

// Direct global -> LDS loads (GLOBAL_LOAD_LDS_DWORDX4 / _DWORD): lane i's 16
// (4) bytes land at M0 + 16 i (4 i).  Written as inline asm so that the
// compiler does not track them: it would otherwise wait for every one of them
// before any LDS read it cannot prove disjoint, and the ring relies on the
// explicit vmcnt waits below instead.  (M0 is not used by any other
// instruction of these kernels.)
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(src), "s"(__builtin_amdgcn_readfirstlane(lds))
               : "memory", "m0");
}
__device__ __forceinline__ void dma4(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
               :
               : "v"(src), "s"(__builtin_amdgcn_readfirstlane(lds))
               : "memory", "m0");
}
// Same loads with a wave-uniform 64-bit base in SGPRs and a 32-bit per-lane
// offset, which keeps the per-step address arithmetic scalar.
__device__ __forceinline__ void dma16_s(uint32_t voff, const void* sbase, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(lds)
               : "memory", "m0");
}
__device__ __forceinline__ void dma4_s(uint32_t voff, const void* sbase, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(lds)
               : "memory", "m0");
}
#pragma clang diagnostic pop

struct Tile {
  const uint8_t* q[2];  // weight / activation codes of the current group
  int64_t ld[2];
  const uint8_t* sc[2];
  int64_t ldsc[2];
  int64_t row0[2];  // first weight / activation row of the tile
  int64_t rows[2];
  int gblk0;        // first block of the group in a scale row
  int nblk;         // K / 32
};

// Issue the DMA of one K step (group G, blocks blk0 .. blk0+nvalid-1) into
// the LDS stage at `st`.
template <int G, int BN, int BM>
__device__ __forceinline__ void issue_step(const Tile& t, uint8_t* st, int blk0, int nvalid) {
  using P = Plan<G, BN, BM>;
  constexpr int CPR = chunks(G);
  constexpr int BB = block_bytes(G);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int valid_bytes = nvalid * BB;
#pragma unroll
  for (int k = 0; k < P::kCodeLoads; ++k) {
    const int inst = wave * P::kCodeLoads + k;  // 64 consecutive 16-byte slots
    const int q = inst * 64 + lane;
    const bool op = q >= BN * CPR;
    const int qq = op ? q - BN * CPR : q;
    const int r = qq / CPR;
    const int c = unswz<G>(qq - r * CPR, r);
    const int64_t nrows = op ? t.rows[1] : t.rows[0];
    int64_t row = (op ? t.row0[1] : t.row0[0]) + r;
    row = row < nrows ? row : nrows - 1;
    const uint8_t* src = (op ? t.q[1] : t.q[0]) + row * (op ? t.ld[1] : t.ld[0]) + blk0 * BB + c * 16;
    src = c * 16 < valid_bytes ? src : kZeroCodes;
    dma16(src, lds_addr(st) + inst * 1024);
  }
  // two aligned scale words per row cover the step's four blocks
  const int off = t.gblk0 + blk0;
  const int a4 = off & ~3;
  const int a4b = a4 + 4 < t.nblk ? a4 + 4 : a4;
#pragma unroll
  for (int k = 0; k < P::kScaleLoads; ++k) {
    const int inst = wave * P::kScaleLoads + k;
    const int d = inst * 64 + lane;
    const int rr = d >> 1;
    const bool op = rr >= BN;
    const int r = op ? rr - BN : rr;
    const int64_t nrows = op ? t.rows[1] : t.rows[0];
    int64_t row = (op ? t.row0[1] : t.row0[0]) + r;
    row = row < nrows ? row : nrows - 1;
    const uint8_t* src = (op ? t.sc[1] : t.sc[0]) + row * (op ? t.ldsc[1] : t.ldsc[0]) + ((d & 1) ? a4b : a4);
    dma4(src, lds_addr(st) + P::kCodeBytes + inst * 256);
  }
}

// Loop-invariant part of a thread's DMA addresses for one group: the byte
// offset of each of its chunks (row * ld + chunk * 16) and scale words
// (row * ldsc + 4 * word) relative to the operand's base pointer.
template <int G, int BN, int BM>
struct DmaPlan {
  using P = Plan<G, BN, BM>;
  uint32_t code[P::kCodeLoads];
  uint32_t scale[P::kScaleLoads];
};

template <int G, int BN, int BM>
__device__ __forceinline__ DmaPlan<G, BN, BM> make_plan(const Tile& t, int wave) {
  using P = Plan<G, BN, BM>;
  constexpr int CPR = chunks(G);
  const int lane = threadIdx.x & 63;
  DmaPlan<G, BN, BM> d;
#pragma unroll
  for (int k = 0; k < P::kCodeLoads; ++k) {
    const int q = (wave * P::kCodeLoads + k) * 64 + lane;
    const bool op = q >= BN * CPR;
    const int qq = op ? q - BN * CPR : q;
    const int r = qq / CPR;
    const int c = unswz<G>(qq - r * CPR, r);
    const int64_t nrows = op ? t.rows[1] : t.rows[0];
    int64_t row = (op ? t.row0[1] : t.row0[0]) + r;
    row = row < nrows ? row : nrows - 1;
    d.code[k] = (uint32_t)(row * (op ? t.ld[1] : t.ld[0])) + c * 16;
  }
#pragma unroll
  for (int k = 0; k < P::kScaleLoads; ++k) {
    const int dd = (wave * P::kScaleLoads + k) * 64 + lane;
    const int rr = dd >> 1;
    const bool op = rr >= BN;
    const int r = op ? rr - BN : rr;
    const int64_t nrows = op ? t.rows[1] : t.rows[0];
    int64_t row = (op ? t.row0[1] : t.row0[0]) + r;
    row = row < nrows ? row : nrows - 1;
    d.scale[k] = (uint32_t)(row * (op ? t.ldsc[1] : t.ldsc[0])) + 4 * (dd & 1);
  }
  return d;
}

// DMA of a full step (four valid blocks whose two scale words lie inside the
// scale row): scalar base pointers, precomputed per-lane offsets.
template <int G, int BN, int BM>
__device__ __forceinline__ void issue_full_step(const Tile& t, const DmaPlan<G, BN, BM>& d, uint32_t st, int wave,
                                                int blk0) {
  using P = Plan<G, BN, BM>;
  constexpr int CPR = chunks(G);
  constexpr int BB = block_bytes(G);
#pragma unroll
  for (int k = 0; k < P::kCodeLoads; ++k) {
    const int inst = wave * P::kCodeLoads + k;
    const bool op = inst * 64 >= BN * CPR;  // uniform: an instruction never spans operands
    dma16_s(d.code[k], (op ? t.q[1] : t.q[0]) + blk0 * BB, st + inst * 1024);
  }
  const int a4 = (t.gblk0 + blk0) & ~3;
#pragma unroll
  for (int k = 0; k < P::kScaleLoads; ++k) {
    const int inst = wave * P::kScaleLoads + k;
    const bool op = inst * 32 >= BN;
    dma4_s(d.scale[k], (op ? t.sc[1] : t.sc[0]) + a4, st + P::kCodeBytes + inst * 256);
  }
}

// One lane's operand fragment for the 32 x 32 x 64 MFMA: tile row `row`,
// 64-channel half kk of the step, lane half g.
template <int G>
__device__ __forceinline__ v8i read_frag(const uint8_t* codes, int row, int kk, int g, int r) {
  constexpr int RB = row_bytes(G);
  const uint8_t* p = codes + row * RB;
  v8i v;
  if constexpr (G == 0) {
    const uint4 d = *reinterpret_cast<const uint4*>(p + 16 * swz<0>(2 * kk + g, r));
    v[0] = (int)d.x;
    v[1] = (int)d.y;
    v[2] = (int)d.z;
    v[3] = (int)d.w;
    v[4] = v[5] = v[6] = v[7] = 0;
  } else if constexpr (G == 1) {
    uint2 d[3];
#pragma unroll
    for (int j = 0; j < 3; ++j) {
      const int b = 24 * (2 * kk + g) + 8 * j;  // logical byte of the piece
      d[j] = *reinterpret_cast<const uint2*>(p + 16 * swz<1>(b >> 4, r) + (b & 15));
    }
    v[0] = (int)d[0].x;
    v[1] = (int)d[0].y;
    v[2] = (int)d[1].x;
    v[3] = (int)d[1].y;
    v[4] = (int)d[2].x;
    v[5] = (int)d[2].y;
    v[6] = v[7] = 0;
  } else {
    const uint4 lo = *reinterpret_cast<const uint4*>(p + 16 * swz<2>(4 * kk + g, r));
    const uint4 hi = *reinterpret_cast<const uint4*>(p + 16 * swz<2>(4 * kk + 2 + g, r));
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

template <int BN, int BM>
using Acc = v16f[BN / 64][BM / 64];

template <int G, int BN, int BM>
__device__ __forceinline__ void compute_step(const uint8_t* st, const uint8_t* one, int off, int nvalid, int wn0,
                                             int wm0, Acc<BN, BM>& acc) {
  using P = Plan<G, BN, BM>;
  constexpr int TN = BN / 64, TM = BM / 64;  // 32-row fragments per wave
  const int lane = threadIdx.x & 63;
  const int g = lane >> 5, r = lane & 31;
  const uint8_t* sc = st + P::kCodeBytes + (off & 3) + g;  // this lane's block in a scale row
  // blocks past the group's end read the constant 1.0 instead (an address
  // select keeps the read unconditional)
  v8i xf[2][TM];
  int xs[2][TM];
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    const bool ok = 2 * kk + g < nvalid;
#pragma unroll
    for (int j = 0; j < TM; ++j) {
      const int row = BN + wm0 + 32 * j + r;
      xf[kk][j] = read_frag<G>(st, row, kk, g, r);
      xs[kk][j] = *(ok ? sc + row * 8 + 2 * kk : one);
    }
  }
  // weight fragments are double-buffered: the next one is read while the
  // MFMAs of the current one run
  v8i wf = read_frag<G>(st, wn0 + r, 0, g, r);
  int ws = *(g < nvalid ? sc + (wn0 + r) * 8 : one);
#pragma unroll
  for (int t = 0; t < 2 * TN; ++t) {
    const int kk = t / TN, i = t % TN;
    v8i wn = wf;
    int wsn = ws;
    if (t + 1 < 2 * TN) {
      const int kn = (t + 1) / TN, in = (t + 1) % TN;
      const int row = wn0 + 32 * in + r;
      wn = read_frag<G>(st, row, kn, g, r);
      wsn = *(2 * kn + g < nvalid ? sc + row * 8 + 2 * kn : one);
    }
#pragma unroll
    for (int j = 0; j < TM; ++j) MM_MFMA32_GROUP(G, acc[i][j], wf, xf[kk][j], ws, xs[kk][j]);
    wf = wn;
    ws = wsn;
  }
}

template <int G, int BN, int BM>
__device__ __forceinline__ void run_group(const GemmArgs& a, uint8_t* lds, int64_t n0, int64_t m0, int wave,
                                          int wn0, int wm0, Acc<BN, BM>& acc) {
  using P = Plan<G, BN, BM>;
  constexpr int NS = P::kStages;
  const int nb = a.nb[G];
  if (nb == 0) return;
  Tile t;
  t.q[0] = a.w.q[G];
  t.q[1] = a.x.q[G];
  t.ld[0] = a.w.ld[G];
  t.ld[1] = a.x.ld[G];
  t.sc[0] = a.w.sc;
  t.sc[1] = a.x.sc;
  t.ldsc[0] = a.w.ldsc;
  t.ldsc[1] = a.x.ldsc;
  t.row0[0] = n0;
  t.row0[1] = m0;
  t.rows[0] = a.w.rows;
  t.rows[1] = a.x.rows;
  t.gblk0 = G == 0 ? 0 : (G == 1 ? a.nb[0] : a.nb[0] + a.nb[1]);
  t.nblk = a.nb[0] + a.nb[1] + a.nb[2];
  const int S = (nb + 3) >> 2;
  auto nval = [&](int s) { return nb - 4 * s < 4 ? nb - 4 * s : 4; };
  const DmaPlan<G, BN, BM> plan = make_plan<G, BN, BM>(t, wave);
  const uint32_t lds0 = lds_addr(lds);
  // full steps take the scalar-address path; a group's last partial step
  // (and a step whose second scale word would pass the row end) the general one
  auto issue = [&](int s) {
    const int b0 = 4 * s;
    uint8_t* st = lds + (s % NS) * P::kStageBytes;
    if (nval(s) == 4 && ((t.gblk0 + b0) & ~3) + 4 < t.nblk)
      issue_full_step<G, BN, BM>(t, plan, lds0 + (s % NS) * P::kStageBytes, wave, b0);
    else
      issue_step<G, BN, BM>(t, st, b0, nval(s));
  };

#pragma unroll
  for (int p = 0; p < NS - 1; ++p)
    if (p < S) issue(p);

  for (int s = 0; s < S; ++s) {
    // steps s+1 .. s+NS-2 may still be in flight; step s must have landed
    if (s + NS - 2 < S) wait_vmcnt<(NS - 2) * P::kLoads>();
    else wait_vmcnt<0>();
    barrier();  // everyone's step-s data is in LDS; everyone is done with step s-1
    // refill the stage that step s-1 used, then multiply step s
    const int sn = s + NS - 1;
    if (sn < S) issue(sn);
    compute_step<G, BN, BM>(lds + (s % NS) * P::kStageBytes, lds + kOneOffset, t.gblk0 + 4 * s, nval(s), wn0,
                            wm0, acc);
  }
  // the next group lays its stages out differently: every wave must be done
  // reading this group's LDS first
  wait_lgkm0();
  barrier();
}

}  // namespace tiled

using namespace tiled;

template <int BN, int BM>
__global__ __launch_bounds__(kThreads, 1) void gemm_tiled_kernel(GemmArgs a, int tiles_n, int tiles_m) {
  extern __shared__ __attribute__((aligned(1024))) uint8_t lds[];
  constexpr int kGroupN = 4;  // weight tiles that share an XCD's L2 at a time

  // workgroup -> tile: consecutive tiles per XCD (workgroups are dealt to the
  // 8 XCDs round-robin), then groups of kGroupN weight tiles, activation
  // tiles fastest inside a group
  const int T = tiles_n * tiles_m;
  const int wg = blockIdx.x;
  const int xcd = wg & 7, k = wg >> 3;
  const int per = T >> 3, extra = T & 7;
  const int t = xcd * per + (xcd < extra ? xcd : extra) + k;
  const int grp = t / (kGroupN * tiles_m);
  const int within = t - grp * kGroupN * tiles_m;
  const int gn = tiles_n - grp * kGroupN < kGroupN ? tiles_n - grp * kGroupN : kGroupN;
  const int tn = grp * kGroupN + within % gn;
  const int tm = within / gn;
  const int64_t n0 = (int64_t)tn * BN, m0 = (int64_t)tm * BM;

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: keeps DMA setup scalar
  const int wn0 = (wave & 1) * (BN / 2);
  const int wm0 = (wave >> 1) * (BM / 2);

  Acc<BN, BM> acc;
#pragma unroll
  for (int i = 0; i < BN / 64; ++i)
#pragma unroll
    for (int j = 0; j < BM / 64; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;
  if (threadIdx.x == 0) lds[kOneOffset] = 127;  // seen after the first barrier

  run_group<0, BN, BM>(a, lds, n0, m0, wave, wn0, wm0, acc);
  run_group<1, BN, BM>(a, lds, n0, m0, wave, wn0, wm0, acc);
  run_group<2, BN, BM>(a, lds, n0, m0, wave, wn0, wm0, acc);

  // lane 32 g + r, register q: output column n = 8 (q/4) + 4 g + q%4 of the
  // fragment, output row m = r
  const int lane = threadIdx.x & 63;
  const int g = lane >> 5, r = lane & 31;
#pragma unroll
  for (int i = 0; i < BN / 64; ++i)
#pragma unroll
    for (int j = 0; j < BM / 64; ++j)
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const v4f c = {acc[i][j][4 * h], acc[i][j][4 * h + 1], acc[i][j][4 * h + 2], acc[i][j][4 * h + 3]};
        store_out4(a, m0 + wm0 + 32 * j + r, n0 + wn0 + 32 * i + 8 * h + 4 * g, c, a.x.rows, a.w.rows);
      }
}

template <int BN, int BM>
static hipError_t launch_tile(const GemmArgs& a, hipStream_t stream) {
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(gemm_tiled_kernel<BN, BM>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBytes);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const int tn = (int)((a.w.rows + BN - 1) / BN), tm = (int)((a.x.rows + BM - 1) / BM);
  hipLaunchKernelGGL((gemm_tiled_kernel<BN, BM>), dim3((unsigned)(tn * tm)), dim3(kThreads), kLdsBytes, stream, a,
                     tn, tm);
  return hipGetLastError();
}

hipError_t launch_gemm_tiled(const GemmArgs& a, hipStream_t stream) {
  // 256 x 256 tiles when they still give every CU several tiles, else
  // 256 x 128 so that the grid covers the 256 CUs
  const int64_t tiles_big = ((a.w.rows + 255) / 256) * ((a.x.rows + 255) / 256);
  if (tiles_big >= 768) return launch_tile<256, 256>(a, stream);
  return launch_tile<256, 128>(a, stream);
}

}  // namespace mm
