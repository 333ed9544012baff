// Mixed MX GEMM for prefill shapes (many activation rows): compute-bound on
// the block-scaled MFMA, so operand tiles are staged in LDS and reused by
// the whole workgroup.
//
// Workgroup tile: BN weight rows (output columns n) x BM activation rows
// (output rows m), four wavefronts in a 2 x 2 grid, each owning a
// (BN/2) x (BM/2) block of 32 x 32 fp32 MFMA accumulators.  The K loop visits
// the E2M1 group, then E3M2, then E4M3 (Sec. 3.1 group order), all
// accumulating into the same registers (Sec. 3.2 "GEMM kernel": one fp32
// accumulation, one bf16 rounding).
//
// Memory pipeline (gfx950): the packed layout stores each 32-row group's
// step contiguously and block-major, so a tile's share of one step is a few
// contiguous runs; it goes straight from global memory into LDS with
// global_load_lds_dwordx4 (1 KB per wavefront instruction, plus one for the
// step's E8M0 scale words), through a ring of as many stages as the tile's
// LDS share (160 KB, or 80 KB for 256 x 128 tiles) holds for the group (a
// stage is a whole layout step, or half of one where whole steps would leave
// fewer than three stages).  Completion is
// tracked with explicit vmcnt waits and bare s_barrier (a __syncthreads fence
// would wait for every load in flight).  The block-major layout makes the
// fragment reads conflict-free: 16 consecutive lanes read 16 consecutive rows
// of one block.
// Workgroups are mapped to tiles XCD by XCD and in groups of weight tiles,
// so the tiles that run together on one XCD share its L2.
#include "gemm_common.hpp"

namespace mm {

namespace tiled {

// LDS per workgroup for TPC workgroups per CU: all 160 KB (TPC = 1), or 80 KB
// (TPC = 2, 256 x 128 tiles only) so that two workgroups share a CU and one's
// pipeline fill and epilogue overlap the other's K loop.  The launch takes
// TPC = 2 when the 256 x 128 tiles outnumber the CUs (measured on 4096 x
// 14336 x 4096: 15 % faster), else the deeper ring of TPC = 1 (8 % faster on
// 2048 x 4096 x 4096, one tile per CU); results are bit-identical.
__host__ __device__ constexpr int lds_bytes(int tpc) { return tpc == 2 ? 80 * 1024 : 160 * 1024; }

// Eight wavefronts per workgroup, two per SIMD (while one waits at a barrier
// or for LDS, the other's MFMAs run), all of them issuing the tile's DMA, in
// a GN x GM grid with 64 activation rows each: 256 x 256 tiles give 128 x 64
// outputs per wavefront (128 accumulator registers), 256 x 128 tiles 64 x 64.
__host__ __device__ constexpr int tile_waves(int, int) { return 8; }
template <int BN, int BM>
struct Shape {
  static constexpr int NW = tile_waves(BN, BM);
  static constexpr int kThreads = 64 * NW;
  static constexpr int WM = 64, GM = BM / WM, GN = NW / GM, WN = BN / GN;  // wavefront grid and tile
  static constexpr int TN = WN / 32, TM = WM / 32;                         // 32-row fragments per wavefront
  static_assert(GN * GM == NW && WN % 32 == 0, "wavefront grid");
};

// Pipeline plan of group G for a BN x BM tile: a "sub-step" is a whole layout
// step (four blocks, two 64-channel slices), or half of one where a whole
// step would leave fewer than three stages in LDS.
template <int G, int BN, int BM, int TPC>
struct Plan {
  static constexpr int RB = step_row_bytes(G);  // bytes per row and layout step
  static constexpr int kRows = BN + BM;
  static constexpr int kLds = lds_bytes(TPC);
  static constexpr int US = kLds / (kRows * (RB + kStepBlocks)) >= 3 ? 1 : 2;  // sub-steps per layout step
  static constexpr int kBlocks = kStepBlocks / US;
  static constexpr int kSlices = kBlocks / 2;
  static constexpr int kGrpBytes = kRowGroup * RB / US;  // one row group, one sub-step
  static constexpr int kWBytes = BN / kRowGroup * kGrpBytes;
  static constexpr int kCodeBytes = kRows / kRowGroup * kGrpBytes;
  static constexpr int kStageBytes = kCodeBytes + kRows * kStepBlocks;  // + the step's scale words
  static constexpr int kStages = kLds / kStageBytes > 8 ? 8 : kLds / kStageBytes;
  static constexpr int kWInstr = kWBytes / 1024;            // DMA instructions carrying weight codes
  static constexpr int NW = Shape<BN, BM>::NW;
  // DMA instruction i (1 KB each) belongs to wavefront i % NW: the first kRem
  // wavefronts issue kCodeLoads of them per sub-step, the others one fewer
  static constexpr int kInstr = kCodeBytes / 1024;
  static constexpr int kCodeLoads = (kInstr + NW - 1) / NW;
  static constexpr int kRem = kInstr % NW;
  static constexpr int kLoads = kCodeLoads + 1;  // + the scale words (most for any wavefront)
  static_assert(kCodeBytes % 1024 == 0 && kWBytes % 1024 == 0, "whole DMA instructions");
  static_assert(kStages >= 3, "ring of at least three stages");
  static_assert((kStages - 2) * kLoads < 64, "vmcnt range");
};

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

template <typename T>
__device__ __forceinline__ T lds_read(uint32_t addr) {
  return *reinterpret_cast<const __attribute__((address_space(3))) T*>((uintptr_t)addr);
}

// Direct global -> LDS load (GLOBAL_LOAD_LDS_DWORDX4) with a wave-uniform
// 64-bit base in SGPRs and a 32-bit per-lane offset: lane i's 16 bytes land
// at M0 + 16 i (M0 is bound as an operand, so the compiler sets it).  Written
// as inline asm so that the compiler does not track the load (it would
// otherwise wait for every one of them before any LDS read it cannot prove
// disjoint); the ring relies on the explicit vmcnt waits.  The s_nop covers
// the wait state between writing M0 and the load reading it.
__device__ __forceinline__ void dma16_s(uint32_t voff, const void* sbase, uint32_t lds) {
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" : : "v"(voff), "s"(sbase), "{m0}"(lds) : "memory");
}

// Per-tile constants of the DMA of one group.
template <int G, int BN, int BM, int TPC>
struct Dma {
  using P = Plan<G, BN, BM, TPC>;
  const uint8_t* code[2];       // weight / activation codes at the tile's first row group
  const uint8_t* sc[2];         // scales at the tile's first row
  int64_t rp[2];                // padded rows of each operand
  uint32_t off[P::kCodeLoads];  // this lane's byte offset for each code instruction
  uint32_t soff;                // this lane's byte offset for the scale instruction
  uint32_t sdst;                // LDS byte offset of this wave's scale words in a stage
  int t0;                       // global layout-step index of the group's first step
};

template <int G, int BN, int BM, int TPC>
__device__ __forceinline__ Dma<G, BN, BM, TPC> make_dma(const GemmArgs& a, int64_t n0, int64_t m0, int wave, int lane) {
  using P = Plan<G, BN, BM, TPC>;
  Dma<G, BN, BM, TPC> d;
  d.rp[0] = a.w.rp;
  d.rp[1] = a.x.rp;
  d.code[0] = a.w.q[G] + n0 * P::RB;
  d.code[1] = a.x.q[G] + m0 * P::RB;
  d.t0 = (G >= 1 ? a.steps[0] : 0) + (G >= 2 ? a.steps[1] : 0);
  // row groups past an operand's padded rows re-read its last row group
  const int last_w = (int)(a.w.rp / kRowGroup - n0 / kRowGroup - 1);
  const int last_x = (int)(a.x.rp / kRowGroup - m0 / kRowGroup - 1);
#pragma unroll
  for (int k = 0; k < P::kCodeLoads; ++k) {
    int inst = k * P::NW + wave;
    inst = inst < P::kInstr ? inst : P::kInstr - 1;  // (not issued)
    const bool op = inst >= P::kWInstr;
    const int q = (inst - (op ? P::kWInstr : 0)) * 1024 + lane * 16;  // byte within the operand's tile slice
    int grp = q / P::kGrpBytes;
    const int within = q - grp * P::kGrpBytes;
    const int last = op ? last_x : last_w;
    grp = grp < last ? grp : last;
    d.off[k] = (uint32_t)(grp * kRowGroup * P::RB + within);
  }
  // scale words: the first half of the wavefronts the weight rows, the
  // second half the activation rows, 4 rows (16 bytes) per lane; rows past
  // the padded rows re-read the last 4
  constexpr int H = P::NW / 2;
  const bool op = wave >= H;
  const int per = op ? BM / H : BN / H;  // rows per wavefront
  const int64_t rp = op ? a.x.rp : a.w.rp;
  const int64_t r0 = op ? m0 : n0;
  int row = (wave % H) * per + lane * 4;  // row within the tile
  row = r0 + row + 4 <= rp ? row : (int)(rp - 4 - r0);
  d.soff = (uint32_t)row * kStepBlocks;
  d.sdst = (uint32_t)(P::kCodeBytes + (op ? BN * kStepBlocks : 0) + (wave % H) * per * kStepBlocks);
  d.sc[0] = a.w.sc + n0 * kStepBlocks;
  d.sc[1] = a.x.sc + m0 * kStepBlocks;
  return d;
}

// Issue the DMA of sub-step p into the LDS stage at byte address st.
template <int G, int BN, int BM, int TPC>
__device__ __forceinline__ void issue(const Dma<G, BN, BM, TPC>& d, uint32_t st, int wave, int lane, int p) {
  using P = Plan<G, BN, BM, TPC>;
  p = __builtin_amdgcn_readfirstlane(p);  // wave-uniform: the bases below must be scalar
  const int64_t s = p / P::US;
  const int u = p % P::US;
  const uint8_t* cw = d.code[0] + s * d.rp[0] * P::RB + u * P::kGrpBytes;
  const uint8_t* cx = d.code[1] + s * d.rp[1] * P::RB + u * P::kGrpBytes;
#pragma unroll
  for (int k = 0; k < P::kCodeLoads; ++k) {
    const int inst = k * P::NW + wave;
    if (P::kRem == 0 || inst < P::kInstr) dma16_s(d.off[k], inst >= P::kWInstr ? cx : cw, st + inst * 1024);
  }
  constexpr int H = P::NW / 2;
  const bool op = wave >= H;
  const int64_t t = d.t0 + s;
  const uint8_t* sb = op ? d.sc[1] + t * d.rp[1] * kStepBlocks : d.sc[0] + t * d.rp[0] * kStepBlocks;
  if (lane < (op ? BM : BN) / H / 4) dma16_s(d.soff, sb, st + d.sdst);
}

// This lane's 32 x 64 fragment at LDS byte address p (block-major record):
// lane 32 g + r holds block g of the slice for E2M1 / E3M2, and channels
// 16g .. 16g+15 of the slice's two blocks for E4M3.
template <int G>
__device__ __forceinline__ v8i read_frag(uint32_t p) {
  v8i v;
  if constexpr (G == 0) {
    const u32x4 d = lds_read<u32x4>(p);
    v[0] = (int)d.x;
    v[1] = (int)d.y;
    v[2] = (int)d.z;
    v[3] = (int)d.w;
    v[4] = v[5] = v[6] = v[7] = 0;
  } else if constexpr (G == 1) {
    const u32x2 d0 = lds_read<u32x2>(p), d1 = lds_read<u32x2>(p + 8), d2 = lds_read<u32x2>(p + 16);
    v[0] = (int)d0.x;
    v[1] = (int)d0.y;
    v[2] = (int)d1.x;
    v[3] = (int)d1.y;
    v[4] = (int)d2.x;
    v[5] = (int)d2.y;
    v[6] = v[7] = 0;
  } else {
    const u32x4 lo = lds_read<u32x4>(p), hi = lds_read<u32x4>(p + 1024);
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
using Acc = v16f[Shape<BN, BM>::TN][Shape<BN, BM>::TM];

// The MFMAs of one sub-step held in the stage at st (layout-step half u).
// All activation fragments of the sub-step are read first; weight fragments
// are double-buffered: the next one is read while the MFMAs of the current
// one run.
template <int G, int BN, int BM, int FS, int TPC>
__device__ __forceinline__ void compute_step(uint32_t st, int u, int wn0, int wm0, Acc<BN, BM>& acc) {
  using P = Plan<G, BN, BM, TPC>;
  constexpr int TN = Shape<BN, BM>::TN, TM = Shape<BN, BM>::TM, SL = P::kSlices;
  constexpr int kSliceOff = G == 0 ? 1024 : (G == 1 ? 1536 : 2048);  // slice 1 starts two blocks on
  const int lane = threadIdx.x & 63;
  const int g = lane >> 5, r = lane & 31;
  const int part = G == 1 ? g * 768 + r * 24 : g * 512 + r * 16;
  const uint32_t bw = st + wn0 / kRowGroup * P::kGrpBytes + part;
  const uint32_t bx = st + P::kWBytes + wm0 / kRowGroup * P::kGrpBytes + part;
  // scale byte of (row, slice kk): block u * kBlocks + 2 kk + g of the layout step
  const uint32_t sw = st + P::kCodeBytes + (wn0 + r) * kStepBlocks + u * P::kBlocks + g;
  const uint32_t sx = st + P::kCodeBytes + (BN + wm0 + r) * kStepBlocks + u * P::kBlocks + g;
  v8i xf[SL][TM];
  int xs[SL][TM];
#pragma unroll
  for (int kk = 0; kk < SL; ++kk)
#pragma unroll
    for (int j = 0; j < TM; ++j) {
      xf[kk][j] = read_frag<G>(bx + j * P::kGrpBytes + kk * kSliceOff);
      xs[kk][j] = lds_read<uint8_t>(sx + j * kRowGroup * kStepBlocks + 2 * kk);
    }
  v8i wf = read_frag<G>(bw);
  int ws = lds_read<uint8_t>(sw);
#pragma unroll
  for (int t = 0; t < SL * TN; ++t) {
    const int kk = t / TN, i = t % TN;
    v8i wn = wf;
    int wsn = ws;
    if (t + 1 < SL * TN) {
      const int kn = (t + 1) / TN, in = (t + 1) % TN;
      wn = read_frag<G>(bw + in * P::kGrpBytes + kn * kSliceOff);
      wsn = lds_read<uint8_t>(sw + in * kRowGroup * kStepBlocks + 2 * kn);
    }
    // keep the next fragment's read ahead of these MFMAs (left alone, the
    // scheduler sinks it below them to reuse the registers, and its latency
    // lands in front of the next MFMA)
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < TM; ++j) MM_MFMA32_GROUP(G, FS, acc[i][j], wf, xf[kk][j], ws, xs[kk][j]);
    wf = wn;
    ws = wsn;
  }
}

// A group's first sub-step issued ahead, during the previous group's last
// one: which group (-1: none) and the ring rotation it was placed with.
struct Ahead {
  int group;
  int rot;
};

// Issue sub-step 0 of group G into a stage of its ring that does not overlap
// the live bytes [live, live + live_bytes) of the group still computing, and
// record the ring rotation that puts it there.
template <int G, int BN, int BM, int TPC>
__device__ __forceinline__ void issue_first(const GemmArgs& a, uint32_t lds0, int64_t n0, int64_t m0, int wave,
                                            uint32_t live, uint32_t live_bytes, Ahead& ah) {
  using P = Plan<G, BN, BM, TPC>;
  int rot = 0;
  for (int k = 0; k < P::kStages; ++k) {
    const uint32_t lo = k * P::kStageBytes, hi = lo + P::kStageBytes;
    if (hi <= live || lo >= live + live_bytes) {
      rot = k;
      break;
    }
  }
  rot = __builtin_amdgcn_readfirstlane(rot);  // uniform; keeps the DMA's M0 value scalar
  const Dma<G, BN, BM, TPC> d = make_dma<G, BN, BM, TPC>(a, n0, m0, wave, threadIdx.x & 63);
  issue<G, BN, BM, TPC>(d, lds0 + rot * P::kStageBytes, wave, threadIdx.x & 63, 0);
  ah.group = G;
  ah.rot = rot;
}

template <int G, int BN, int BM, int FS, int TPC>
__device__ __forceinline__ void run_group(const GemmArgs& a, uint32_t lds0, int64_t n0, int64_t m0, int wave,
                                          int wn0, int wm0, Acc<BN, BM>& acc, Ahead& ah) {
  using P = Plan<G, BN, BM, TPC>;
  constexpr int NS = P::kStages;
  const int S = a.steps[G];
  if (S == 0) return;
  const int PS = S * P::US;  // sub-steps
  const int lane = threadIdx.x & 63;
  const Dma<G, BN, BM, TPC> d = make_dma<G, BN, BM, TPC>(a, n0, m0, wave, lane);
  // sub-step q lives in stage (q + rot) % NS; sub-step 0 may already be in
  // flight (issued during the previous group's last sub-step)
  const bool first_ahead = ah.group == G;
  const int rot = __builtin_amdgcn_readfirstlane(first_ahead ? ah.rot : 0);
  auto stage = [&](int q) { return lds0 + (uint32_t)__builtin_amdgcn_readfirstlane(((q + rot) % NS) * P::kStageBytes); };

  for (int q = first_ahead ? 1 : 0; q < NS - 1; ++q)
    if (q < PS) issue<G, BN, BM, TPC>(d, stage(q), wave, lane, q);

  for (int p = 0; p < PS; ++p) {
    // sub-steps p+1 .. p+NS-2 may still be in flight; sub-step p must have
    // landed
    if (p + NS - 2 < PS) {
      if (P::kRem == 0 || wave < P::kRem)
        wait_vmcnt<(NS - 2) * P::kLoads>();
      else
        wait_vmcnt<(NS - 2) * (P::kLoads - 1)>();
    } else {
      wait_vmcnt<0>();
    }
    barrier();  // everyone's sub-step-p data is in LDS; everyone is done with p-1
    // refill the stage that sub-step p-1 used; during the last sub-step,
    // start the next non-empty group instead
    if (p + NS - 1 < PS) {
      issue<G, BN, BM, TPC>(d, stage(p + NS - 1), wave, lane, p + NS - 1);
    } else if (p == PS - 1) {
      const uint32_t live = ((p + rot) % NS) * P::kStageBytes;
      if constexpr (G < 2) {
        if (a.steps[G + 1] > 0)
          issue_first<G + 1, BN, BM, TPC>(a, lds0, n0, m0, wave, live, P::kStageBytes, ah);
        else if constexpr (G == 0) {
          if (a.steps[2] > 0) issue_first<2, BN, BM, TPC>(a, lds0, n0, m0, wave, live, P::kStageBytes, ah);
        }
      }
    }
    compute_step<G, BN, BM, FS, TPC>(stage(p), p % P::US, wn0, wm0, acc);
  }
  // the next group lays its stages out differently: every wave must be done
  // reading this group's LDS first
  wait_lgkm0();
  barrier();
}

}  // namespace tiled

using namespace tiled;

template <int BN, int BM, int FS, int TPC>
__global__ __launch_bounds__(64 * tile_waves(BN, BM), TPC) void gemm_tiled_kernel(GemmArgs a, int tiles_n,
                                                                                                     int tiles_m) {
  using SH = Shape<BN, BM>;
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
  const int wn0 = (wave % SH::GN) * SH::WN;
  const int wm0 = (wave / SH::GN) * SH::WM;
  const uint32_t lds0 = lds_addr(lds);

  Acc<BN, BM> acc;
#pragma unroll
  for (int i = 0; i < SH::TN; ++i)
#pragma unroll
    for (int j = 0; j < SH::TM; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;

  Ahead ah{-1, 0};
  run_group<0, BN, BM, FS, TPC>(a, lds0, n0, m0, wave, wn0, wm0, acc, ah);
  run_group<1, BN, BM, FS, TPC>(a, lds0, n0, m0, wave, wn0, wm0, acc, ah);
  run_group<2, BN, BM, FS, TPC>(a, lds0, n0, m0, wave, wn0, wm0, acc, ah);

  // Epilogue: the bf16 tile is assembled in LDS (free again after the last
  // group's closing barrier) and written out as whole rows, 16 bytes per
  // lane, so every store fills full cache lines.  Lane 32 g + r, register q
  // holds output column n = 8 (q/4) + 4 g + q%4 of its fragment and output
  // row m = r.  Rows are padded by 16 bytes: the fragment writes of 32 lanes
  // (32 rows) then fall on distinct banks.
  constexpr int kRowStride = BN * 2 + 16;
  static_assert(BM * kRowStride <= lds_bytes(TPC), "epilogue tile fits LDS");
  const int lane = threadIdx.x & 63;
  const int g = lane >> 5, r = lane & 31;
#pragma unroll
  for (int i = 0; i < SH::TN; ++i)
#pragma unroll
    for (int j = 0; j < SH::TM; ++j)
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const uint32_t lo = f32_to_bf16_rne(acc[i][j][4 * h]) | (f32_to_bf16_rne(acc[i][j][4 * h + 1]) << 16);
        const uint32_t hi = f32_to_bf16_rne(acc[i][j][4 * h + 2]) | (f32_to_bf16_rne(acc[i][j][4 * h + 3]) << 16);
        const uint32_t at = lds0 + (wm0 + 32 * j + r) * kRowStride + (wn0 + 32 * i + 8 * h + 4 * g) * 2;
        *reinterpret_cast<__attribute__((address_space(3))) u32x2*>((uintptr_t)at) = u32x2{lo, hi};
      }
  __syncthreads();
  constexpr int kChunks = BN / 8;  // 16-byte chunks per row
  const int64_t M = a.x.rows, N = a.w.rows;
  for (int c = threadIdx.x; c < BM * kChunks; c += SH::kThreads) {
    const int row = c / kChunks, col = (c - row * kChunks) * 8;
    const int64_t m = m0 + row, n = n0 + col;
    if (m >= M || n >= N) continue;
    const u32x4 v = lds_read<u32x4>(lds0 + row * kRowStride + col * 2);
    uint16_t* dst = a.y + m * a.ldy + n;
    if (n + 8 <= N) {
      *reinterpret_cast<u32x4*>(dst) = v;
    } else {
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
      for (int q = 0; q < (int)(N - n); ++q) dst[q] = (uint16_t)(w[q >> 1] >> (16 * (q & 1)));
    }
  }
}

template <int BN, int BM, int FS, int TPC>
static hipError_t launch_tile_fs(const GemmArgs& a, hipStream_t stream) {
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(gemm_tiled_kernel<BN, BM, FS, TPC>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes(TPC));
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const int tn = (int)((a.w.rows + BN - 1) / BN), tm = (int)((a.x.rows + BM - 1) / BM);
  hipLaunchKernelGGL((gemm_tiled_kernel<BN, BM, FS, TPC>), dim3((unsigned)(tn * tm)), dim3(Shape<BN, BM>::kThreads),
                     lds_bytes(TPC), stream, a,
                     tn, tm);
  return hipGetLastError();
}

// The format set is an instruction immediate: one kernel per set.
template <int BN, int BM, int TPC>
static hipError_t launch_tile(const GemmArgs& a, hipStream_t stream) {
  switch (a.fs) {
    case 0: return launch_tile_fs<BN, BM, 0, TPC>(a, stream);
    case 1: return launch_tile_fs<BN, BM, 1, TPC>(a, stream);
    case 2: return launch_tile_fs<BN, BM, 2, TPC>(a, stream);
    case 3: return launch_tile_fs<BN, BM, 3, TPC>(a, stream);
  }
  return hipErrorInvalidValue;
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

hipError_t launch_gemm_tiled(const GemmArgs& a, hipStream_t stream) {
  // 256 x 256 tiles when they still give every CU several tiles, else
  // 256 x 128 (twice the tiles), two per CU when they outnumber the CUs
  const int64_t t256 = ((a.w.rows + 255) / 256) * ((a.x.rows + 255) / 256);
  if (t256 >= 768) return launch_tile<256, 256, 1>(a, stream);
  int cus = 0;
  hipError_t e = device_cus(&cus);
  if (e != hipSuccess) return e;
  const int64_t t128 = ((a.w.rows + 255) / 256) * ((a.x.rows + 127) / 128);
  if (t128 > cus) return launch_tile<256, 128, 2>(a, stream);
  return launch_tile<256, 128, 1>(a, stream);
}

}  // namespace mm
