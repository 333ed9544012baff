// Mixed MX GEMM for prefill shapes (many activation rows): compute-bound on
// the block-scaled MFMA, so operand tiles are staged in LDS and reused by the
// whole workgroup.
//
// Workgroup tile: BN = 256 weight rows (output columns n) x BM = 256 or 128
// activation rows (output rows m).  Four wavefronts, one per SIMD, in a
// 2 x 2 grid; each owns a (BN/2) x (BM/2) block of 32 x 32 fp32 MFMA
// accumulators (128 x 128: 256 accumulator registers, in the AGPR half of
// the register file).  A wavefront reads TN + TM operand fragments per
// 64-channel slice for TN * TM MFMAs, half the LDS traffic per MFMA of
// 128 x 64 blocks.  The K loop visits the E2M1 group, then E3M2, then E4M3
// (Sec. 3.1 group order), all accumulating into the same registers
// (Sec. 3.2 "GEMM kernel": one fp32 accumulation, one bf16 rounding at the
// end).
//
// Memory pipeline (gfx950): the packed layout stores each 32-row group's
// layout step contiguously and block-major, so a tile's share of a step is
// a few contiguous runs; it goes straight from global memory into LDS with
// global_load_lds_dwordx4 (1 KB per wavefront instruction).  One ring of
// equal slots serves all three groups: a slot holds one "stage", an E2M1
// layout step (128 channels, two slices) or half an E3M2 / E4M3 step (64
// channels, one slice), plus the step's E8M0 scale words of every tile row.
// The ring runs on across group boundaries, so the next group's first
// stages are in flight while the current group finishes.
//
// Every wavefront issues the same number of loads for every stage: eight
// 1 KB code loads (wavefronts 0-1 the weight rows, 2-3 the activation rows;
// a share smaller than eight loads is completed by loading its last pieces
// again, into the same LDS bytes with the same data) and one scale load.
// The vmcnt wait for a stage is then one constant, and issuing the next
// stage is a loop-carried cursor (one base pointer per wavefront, per-lane
// offsets fixed per group) instead of per-stage address arithmetic, which
// a single wavefront per SIMD could not hide behind its MFMAs.  The K loop
// runs in segments whose refills stay in one group: inside a segment the
// cursor only adds a precomputed increment (no branch, its per-lane offsets
// untouched), and it is re-pointed between segments; with the group change
// tested every stage, the scalar bookkeeping of a stage outweighed its
// MFMAs (5-10 % slower).
//
// Per stage q: wait for this wavefront's LDS reads and for its loads of
// stage q+1, one s_barrier (everyone's part of stage q+1 has landed and
// every read of stage q's slot is done); then the stage's MFMAs, each
// followed by its share of the other work: the loads that refill stage q's
// slot with stage q + slots, and the LDS reads of stage q+1's operands.
// The sched_barrier fences keep that order.  Workgroups are mapped to tiles
// XCD by XCD and in groups of weight tiles, so the tiles that run together
// on one XCD share its L2.
#include "gemm_common.hpp"

namespace mm {

namespace tiled {

constexpr int kLdsBytes = 160 * 1024;
constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kCodeLoads = 8;  // code loads per wavefront and stage
constexpr int kLoads = kCodeLoads + 1;  // + the scale load

// A stage of group G: E2M1 one layout step (two 64-channel slices), E3M2 and
// E4M3 half a step (one slice).
__host__ __device__ constexpr int stage_slices(int G) { return G == 0 ? 2 : 1; }
// Bytes of one 32-row group's share of a stage.
__host__ __device__ constexpr int stage_grp_bytes(int G) { return G == 1 ? 1536 : 2048; }
// LDS read pattern of a group: 0 for the 2 KB row-group shares of E2M1 and
// E4M3 (their fragment reads are the same), 1 for the 1.5 KB ones of E3M2.
__host__ __device__ constexpr int pattern(int G) { return G == 1 ? 1 : 0; }

template <int BN, int BM>
struct Tile {
  static constexpr int WN = BN / 2, WM = BM / 2;    // a wavefront's block
  static constexpr int TN = WN / 32, TM = WM / 32;  // its 32-row fragments
  static constexpr int F = TN + TM;
  static constexpr int kRows = BN + BM;
  static constexpr int kScaleOff = kRows * 64;  // scale words follow the largest code payload (64 B per row)
  static constexpr int kSlotBytes = kScaleOff + kRows * kStepBlocks;
  // four slots for both shapes: the 256 x 128 tile fits six, but with four
  // its K loop starts after four stages instead of six and it measured 2-4 %
  // faster (2048 x 4096 x 4096: 30.8 -> 30.1 us)
  static constexpr int kSlots = 4;
  static_assert(BN == 256 && (BM == 256 || BM == 128), "tile shapes");
  static_assert(kSlots * kSlotBytes <= kLdsBytes, "the ring fits LDS");
  static_assert((kSlots - 1) * kLoads < 64, "vmcnt range");
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

// The same for part of the lanes: the exec mask is narrowed inside the asm
// statement (and restored before it ends), so a partial load stays one
// straight-line instruction that the vmcnt bookkeeping counts once.
__device__ __forceinline__ void dma16_masked(uint32_t voff, const void* sbase, uint32_t lds, uint64_t mask) {
  uint64_t saved;
  asm volatile(
      "s_mov_b64 %0, exec\n\t"
      "s_mov_b64 exec, %4\n\t"
      "s_nop 1\n\t"
      "global_load_lds_dwordx4 %1, %2\n\t"
      "s_mov_b64 exec, %0"
      : "=&s"(saved)
      : "v"(voff), "s"(sbase), "{m0}"(lds), "s"(mask)
      : "memory");
}

// A wave-uniform value kept in SGPRs (the compiler is told it is uniform).
__device__ __forceinline__ uint32_t uni(uint32_t v) { return (uint32_t)__builtin_amdgcn_readfirstlane((int)v); }
__device__ __forceinline__ const uint8_t* uni(const uint8_t* p) {
  const uint64_t v = (uint64_t)p;
  const uint64_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
  const uint64_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(v >> 32));
  return (const uint8_t*)(lo | (hi << 32));
}

// Hide a value from loop-invariant code motion (hoisting every derived
// address out of the K loop would keep them all live across it).
template <typename V>
__device__ __forceinline__ V opaque_s(V v) {
  asm volatile("" : "+s"(v));
  return v;
}

// ---------------------------------------------------------------------------
// DMA cursor: where the next stage to issue comes from and goes to.
// ---------------------------------------------------------------------------

// Per-tile constants of this wavefront's loads.
struct DmaConst {
  const uint8_t* code0;    // this wavefront's operand codes at the tile's first row, per group
  const uint8_t* code1;
  const uint8_t* code2;
  int64_t rstride0;        // bytes between layout steps of a group (padded rows x step row bytes)
  int64_t rstride1;
  int64_t rstride2;
  const uint8_t* sc;       // this wavefront's operand scales at the tile's first row, layout step 0
  int64_t sstride;         // bytes between layout steps of the scales
  uint32_t soff;           // this lane's byte offset for the scale load
  uint32_t sdst;           // LDS offset of this wavefront's scale words in a slot
  uint64_t smask;          // lanes that take part in the scale load
  int last;                // last row group (relative to the tile) with rows, of this wavefront's operand
  int rows_op;             // tile rows of this wavefront's operand (BN or BM)
  int op;                  // 0: weight rows, 1: activation rows
  int half;                // which half of the operand's share this wavefront loads
  uint32_t op_lds;         // LDS offset of the operand's codes in a slot (2 KB row-group shares)
  uint32_t op_lds6;        // the same for 1.5 KB shares
};

// The state that advances stage by stage.
struct DmaCursor {
  const uint8_t* bc;  // code base of the next stage to issue
  const uint8_t* bs;  // scale base of the next stage to issue
  int q;              // its stage index (it stays on the last stage: later issues repeat it)
  int g;              // its group
  int u;              // its half of the layout step (E3M2 / E4M3)
  // the step to the next stage inside a segment (see run_group): code and
  // scale base increments when u is 0 / 1, and whether u alternates
  int64_t inc0, inc1, sinc0, sinc1;
  int flip;
  uint32_t doff[kCodeLoads];  // this lane's global byte offset for each code load of group g
  uint32_t mo[kCodeLoads];    // LDS offset (in a slot) of each code load of group g
};

// Per-lane offsets of group G's code loads for this wavefront.
template <int G>
__device__ __forceinline__ void group_offsets(const DmaConst& k, DmaCursor& cur, int lane) {
  constexpr int GB = stage_grp_bytes(G);
  constexpr int RB = step_row_bytes(G);
  const int n = k.rows_op / kRowGroup * GB / 1024;  // 1 KB loads of the operand's share
  const int per = n / 2;                              // of which this wavefront's half
  const uint32_t base_lds = G == 1 ? k.op_lds6 : k.op_lds;
#pragma unroll
  for (int p = 0; p < kCodeLoads; ++p) {
    const int li = k.half * per + p % per;  // load within the operand's share (repeats past `per`)
    const int x = li * 1024 + lane * 16;     // this lane's byte within the share
    int grp = x / GB;
    const int within = x - grp * GB;
    grp = grp < k.last ? grp : k.last;  // row groups past the padded rows re-read the last one
    cur.doff[p] = (uint32_t)(grp * kRowGroup * RB + within);
    cur.mo[p] = uni(base_lds + (uint32_t)li * 1024u);
  }
}

// Stage boundaries: group 0 is [0, q1), group 1 [q1, q2), group 2 [q2, Q);
// t1, t2 the first layout steps of groups 1 and 2 in the scale buffer.
struct Stages {
  int q1, q2, Q, t1, t2;
};

__device__ __forceinline__ int stage_group(const Stages& S, int q) { return q < S.q1 ? 0 : (q < S.q2 ? 1 : 2); }

// Point the cursor at the first stage of group g (global stage index q).
__device__ __forceinline__ void cursor_group(const DmaConst& k, const Stages& S, DmaCursor& cur, int g, int q,
                                             int lane) {
  cur.g = g;
  cur.q = q;
  cur.u = 0;
  if (g == 0)
    cur.bc = uni(k.code0);
  else if (g == 1)
    cur.bc = uni(k.code1);
  else
    cur.bc = uni(k.code2);
  cur.bs = uni(k.sc + (int64_t)(g == 0 ? 0 : (g == 1 ? S.t1 : S.t2)) * k.sstride);
  if (g == 0)
    group_offsets<0>(k, cur, lane);
  else if (g == 1)
    group_offsets<1>(k, cur, lane);
  else
    group_offsets<2>(k, cur, lane);
}

// Advance the cursor past the stage it points at (it stays on the last
// stage once there).
__device__ __forceinline__ void cursor_next(const DmaConst& k, const Stages& S, DmaCursor& cur, int lane) {
  const int nq = cur.q + 1;
  if (nq >= S.Q) return;
  const int ng = stage_group(S, nq);
  if (ng != cur.g) {
    cursor_group(k, S, cur, ng, nq, lane);
    return;
  }
  cur.q = nq;
  if (cur.g == 0) {
    cur.bc += k.rstride0;
    cur.bs += k.sstride;
  } else if (cur.u == 0) {
    cur.bc += cur.g == 1 ? stage_grp_bytes(1) : stage_grp_bytes(2);
    cur.u = 1;
  } else {
    if (cur.g == 1)
      cur.bc += k.rstride1 - stage_grp_bytes(1);
    else
      cur.bc += k.rstride2 - stage_grp_bytes(2);
    cur.bs += k.sstride;
    cur.u = 0;
  }
  cur.bc = uni(cur.bc);
  cur.bs = uni(cur.bs);
}

// Point the cursor at stage qr for a run of stages whose refills stay in
// qr's group (hold = true: every refill of the run is qr itself, the last
// stage).  Only here do the group's per-lane offsets change.
__device__ __forceinline__ void cursor_segment(const DmaConst& k, const Stages& S, DmaCursor& cur, int qr, bool hold,
                                               int lane) {
  const int g = stage_group(S, qr);
  cursor_group(k, S, cur, g, qr, lane);  // the group's first stage, u = 0
  if (g == 0) {
    cur.bc = uni(cur.bc + (int64_t)qr * k.rstride0);
    cur.bs = uni(cur.bs + (int64_t)qr * k.sstride);
    cur.inc0 = cur.inc1 = k.rstride0;
    cur.sinc0 = cur.sinc1 = k.sstride;
    cur.flip = 0;
  } else {
    const int s = qr - (g == 1 ? S.q1 : S.q2);
    const int64_t rs = g == 1 ? k.rstride1 : k.rstride2;
    const int64_t gb = g == 1 ? stage_grp_bytes(1) : stage_grp_bytes(2);
    cur.bc = uni(cur.bc + (int64_t)(s >> 1) * rs + (s & 1) * gb);
    cur.bs = uni(cur.bs + (int64_t)(s >> 1) * k.sstride);
    cur.u = s & 1;
    cur.inc0 = gb;
    cur.inc1 = rs - gb;
    cur.sinc0 = 0;
    cur.sinc1 = k.sstride;
    cur.flip = 1;
  }
  if (hold) {
    cur.inc0 = cur.inc1 = cur.sinc0 = cur.sinc1 = 0;
    cur.flip = 0;
  }
}

// One stage on inside a segment: no branch, the offsets untouched.
__device__ __forceinline__ void cursor_step(DmaCursor& cur) {
  cur.bc = uni(cur.bc + (cur.u ? cur.inc1 : cur.inc0));
  cur.bs = uni(cur.bs + (cur.u ? cur.sinc1 : cur.sinc0));
  cur.u ^= cur.flip;
}

// Load P of the stage the cursor points at, into the slot at LDS byte
// address st: code loads 0..7, then the scale load (P = 8).
template <int P>
__device__ __forceinline__ void issue_load(const DmaConst& k, const DmaCursor& cur, uint32_t st) {
  if constexpr (P < kCodeLoads)
    dma16_s(cur.doff[P], cur.bc, st + cur.mo[P]);
  else
    dma16_masked(k.soff, cur.bs, st + k.sdst, k.smask);
}

template <int P = 0>
__device__ __forceinline__ void issue_all(const DmaConst& k, const DmaCursor& cur, uint32_t st) {
  if constexpr (P < kLoads) {
    issue_load<P>(k, cur, st);
    issue_all<P + 1>(k, cur, st);
  }
}

// ---------------------------------------------------------------------------
// Operands in registers and the MFMAs.
// ---------------------------------------------------------------------------

// Registers of one stage's operands, any group: TN weight then TM
// activation fragments of 8 dwords, and the raw scale words of their rows
// in the same order.  E2M1: dwords 0-3 hold the stage's first 64-channel
// slice and 4-7 its second; E3M2: dwords 0-5; E4M3: all 8.
template <int BN, int BM>
struct Ops {
  v8i f[Tile<BN, BM>::F];
  int s[Tile<BN, BM>::F];
};

// LDS byte addresses of one stage's reads for this lane.
struct OpsAddr {
  uint32_t w, x, sw, sx;
};

template <int PT, int BN, int BM>
__device__ __forceinline__ OpsAddr ops_addr(uint32_t st, int wn0, int wm0, int lane) {
  using T = Tile<BN, BM>;
  constexpr int GB = PT == 0 ? 2048 : 1536;
  constexpr int kWBytes = BN / kRowGroup * GB;
  const int g = lane >> 5, r = lane & 31;
  const int part = PT == 0 ? g * 512 + r * 16 : g * 768 + r * 24;
  OpsAddr ad;
  ad.w = st + wn0 / kRowGroup * GB + part;
  ad.x = st + kWBytes + wm0 / kRowGroup * GB + part;
  ad.sw = st + T::kScaleOff + (wn0 + r) * kStepBlocks;
  ad.sx = st + T::kScaleOff + (BN + wm0 + r) * kStepBlocks;
  return ad;
}

// This lane's fragment at LDS byte address p (block-major record).
// Pattern 0: lane 32 g + r reads 16 bytes of block g and 16 of block 2 + g
// (E2M1: block g of each slice; E4M3: channels 16g .. 16g+15 of each of the
// slice's two blocks).  Pattern 1 (E3M2): the 24 bytes of block g.
template <int PT>
__device__ __forceinline__ void read_frag(v8i& v, uint32_t p) {
  if constexpr (PT == 0) {
    const u32x4 lo = lds_read<u32x4>(p), hi = lds_read<u32x4>(p + 1024);
    v = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
  } else {
    const u32x2 d0 = lds_read<u32x2>(p), d1 = lds_read<u32x2>(p + 8), d2 = lds_read<u32x2>(p + 16);
    v[0] = (int)d0.x;
    v[1] = (int)d0.y;
    v[2] = (int)d1.x;
    v[3] = (int)d1.y;
    v[4] = (int)d2.x;
    v[5] = (int)d2.y;
  }
}

// Read item I of a stage into o: the scale words of the weight rows and of
// the activation rows first (they are needed first), then weight fragments
// 0..TN-1 and activation fragments.
template <int PT, int I, int BN, int BM>
__device__ __forceinline__ void read_item(Ops<BN, BM>& o, const OpsAddr& ad) {
  using T = Tile<BN, BM>;
  constexpr int GB = PT == 0 ? 2048 : 1536;
  if constexpr (I < T::F) {
    if constexpr (I < T::TN) o.s[I] = lds_read<int>(ad.sw + I * kRowGroup * kStepBlocks);
    else o.s[I] = lds_read<int>(ad.sx + (I - T::TN) * kRowGroup * kStepBlocks);
  } else {
    constexpr int f = I - T::F;
    if constexpr (f < T::TN) read_frag<PT>(o.f[f], ad.w + f * GB);
    else read_frag<PT>(o.f[f], ad.x + (f - T::TN) * GB);
  }
}

template <int PT, int I0, int I1, int BN, int BM>
__device__ __forceinline__ void read_items(Ops<BN, BM>& o, const OpsAddr& ad) {
  if constexpr (I0 < I1) {
    read_item<PT, I0>(o, ad);
    read_items<PT, I0 + 1, I1>(o, ad);
  }
}

template <int BN, int BM>
using Acc = v16f[Tile<BN, BM>::TN][Tile<BN, BM>::TM];

// The MFMA operand of one slice of a fragment.
template <int G, int KK>
__device__ __forceinline__ v8i operand(const v8i& f) {
  if constexpr (G == 0) return KK == 0 ? v8i{f[0], f[1], f[2], f[3], 0, 0, 0, 0} : v8i{f[4], f[5], f[6], f[7], 0, 0, 0, 0};
  else if constexpr (G == 1) return v8i{f[0], f[1], f[2], f[3], f[4], f[5], 0, 0};
  else return f;
}

// Loads P0 .. P1-1 of the refill.
template <int P0, int P1>
__device__ __forceinline__ void issue_loads(const DmaConst& k, const DmaCursor& cur, uint32_t st) {
  if constexpr (P0 < P1) {
    issue_load<P0>(k, cur, st);
    issue_loads<P0 + 1, P1>(k, cur, st);
  }
}

// Everything a stage does beside its MFMAs.
struct StageWork {
  uint32_t st_refill;  // slot being refilled (stage q's)
  OpsAddr ad;          // reads of stage q+1
};

// The MFMAs of one group-G stage (acc += W x X^T), in program order: E2M1
// runs its first slice over every accumulator, then its second (so no MFMA
// waits for the one before it).  Lane 32 g + r needs the scale of block
// 2 kk' + g of its row, kk' the slice's 64-channel position in the layout
// step: sc holds the scale words shifted right by 8 g (+ 16 for the second
// half of an E3M2 / E4M3 step) and op_sel picks byte 2 kk (kk the slice
// within the stage).  Each MFMA is followed by its share of the refill's
// loads (all kLoads of them spread over the stage's MFMAs, however many
// there are) and of the reads of the next stage (pattern PN, spread over the
// first three quarters of the MFMAs so that they have landed when the next
// stage starts).
template <int G, int PN, int FS, int T, int BN, int BM>
__device__ __forceinline__ void mfma_block(Acc<BN, BM>& acc, const Ops<BN, BM>& o, const int* sc, Ops<BN, BM>& nxt,
                                           const DmaConst& k, const DmaCursor& cur, const StageWork& w) {
  constexpr int TN = Tile<BN, BM>::TN, TM = Tile<BN, BM>::TM;
  constexpr int kPer = TN * TM;
  constexpr int kM = stage_slices(G) * kPer;
  if constexpr (T < kM) {
    constexpr int fmt = group_fmt(G, FS);
    constexpr int KK = T / kPer, i = (T % kPer) / TM, j = T % TM;
    acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(operand<G, KK>(o.f[i]), operand<G, KK>(o.f[TN + j]),
                                                                acc[i][j], fmt, fmt, 2 * KK, sc[i], 2 * KK, sc[TN + j]);
    issue_loads<(T * kLoads + kM - 1) / kM, ((T + 1) * kLoads + kM - 1) / kM>(k, cur, w.st_refill);
    constexpr int kSpan = kM * 3 / 4;
    constexpr int kItems = 2 * Tile<BN, BM>::F;
    if constexpr (T < kSpan) read_items<PN, T * kItems / kSpan, (T + 1) * kItems / kSpan>(nxt, w.ad);
    __builtin_amdgcn_sched_barrier(0);
    mfma_block<G, PN, FS, T + 1>(acc, o, sc, nxt, k, cur, w);
  }
}

// Kernel-wide state of one tile.
template <int BN, int BM>
struct Ctx {
  DmaConst k;
  Stages S;
  uint32_t lds0;
  int wn0, wm0, lane;
};

// Stage q of group G: its operands are in `cur`, stage q+1's are read into
// `nxt` (with group G's pattern: for the group's last stage those reads are
// of no use, harmlessly, and the next group reads its first stage again).
template <int G, int FS, int BN, int BM>
__device__ __forceinline__ void stage(const Ctx<BN, BM>& c, Acc<BN, BM>& acc, DmaCursor& dc, uint32_t& st, int q,
                                      const Ops<BN, BM>& cur, Ops<BN, BM>& nxt) {
  using T = Tile<BN, BM>;
  constexpr int NS = T::kSlots;
  const Stages& S = c.S;
  // scale operands: shift by 8 g, + 16 for the second half of an E3M2 / E4M3 step
  const int u = G == 0 ? 0 : ((q - (G == 1 ? S.q1 : S.q2)) & 1);
  const int shift = 8 * (c.lane >> 5) + 16 * u;
  int sc[T::F];
#pragma unroll
  for (int f = 0; f < T::F; ++f) sc[f] = (int)((uint32_t)cur.s[f] >> shift);
  // stage q+1 landed (this wavefront's loads: every stage issues kLoads, and
  // the NS - 2 stages after q+1 may still be in flight), everyone's reads of
  // stage q's slot are done
  wait_lgkm0();
  wait_vmcnt<(NS - 2) * kLoads>();
  barrier();
  const uint32_t st_end = c.lds0 + NS * T::kSlotBytes;
  const uint32_t st_next = st + T::kSlotBytes < st_end ? st + T::kSlotBytes : c.lds0;
  StageWork w;
  w.st_refill = __builtin_amdgcn_readfirstlane(st);
  w.ad = ops_addr<pattern(G), BN, BM>(st_next, opaque_s(c.wn0), opaque_s(c.wm0), c.lane);
  // the cursor moves on before the MFMAs (straight-line: a branch there
  // would end the MFMAs' basic block and let them sink away from the work
  // they are interleaved with); this stage's refill uses the position it had
  const DmaCursor issue = dc;
  cursor_step(dc);
  mfma_block<G, pattern(G), FS, 0>(acc, cur, sc, nxt, c.k, issue, w);
  st = st_next;
}

// All stages of group G, two per iteration (the operand registers
// alternate).  On entry the group's first stage has landed and every
// wavefront has passed the barrier after it, and st is its slot; on exit
// the same holds for the next group's first stage.
template <int G, int FS, int BN, int BM>
__device__ __forceinline__ void run_group(const Ctx<BN, BM>& c, Acc<BN, BM>& acc, DmaCursor& dc, uint32_t& st) {
  using T = Tile<BN, BM>;
  const int qb = G == 0 ? 0 : (G == 1 ? c.S.q1 : c.S.q2);
  const int qe = G == 0 ? c.S.q1 : (G == 1 ? c.S.q2 : c.S.Q);
  if (qb == qe) return;
  constexpr int NS = T::kSlots;
  const Stages& S = c.S;
  Ops<BN, BM> A, B;
  read_items<pattern(G), 0, 2 * T::F>(A, ops_addr<pattern(G), BN, BM>(st, c.wn0, c.wm0, c.lane));
  // segments: runs of stages whose refills (stage q + NS, the last one
  // again past the end) stay in one group, so that inside a run the cursor
  // only steps; it is re-pointed between runs
  int q = qb;
  while (q < qe) {
    const int qr = q + NS < S.Q ? q + NS : S.Q - 1;
    const bool hold = q + NS >= S.Q - 1;
    int e = qe;
    if (!hold) {
      const int gr = stage_group(S, qr);
      if (gr == 0 && S.q1 - NS < e) e = S.q1 - NS;
      if (gr <= 1 && S.q2 - NS < e) e = S.q2 - NS;
      if (S.Q - 1 - NS < e) e = S.Q - 1 - NS;
    }
    e = e > q ? e : q + 1;
    cursor_segment(c.k, S, dc, qr, hold, c.lane);
    for (; q + 1 < e; q += 2) {
      stage<G, FS>(c, acc, dc, st, q, A, B);
      stage<G, FS>(c, acc, dc, st, q + 1, B, A);
    }
    if (q < e) {
      stage<G, FS>(c, acc, dc, st, q, A, B);
      A = B;  // the next run starts from A
      ++q;
    }
  }
}

}  // namespace tiled

using namespace tiled;

template <int BN, int BM, int FS>
__global__ __launch_bounds__(kThreads, 1) void gemm_tiled_kernel(GemmArgs a, int tiles_n, int tiles_m) {
  using T = Tile<BN, BM>;
  constexpr int NS = T::kSlots;
  extern __shared__ __attribute__((aligned(1024))) uint8_t lds[];
  constexpr int kGroupN = 4;  // weight tiles that share an XCD's L2 at a time

  // workgroup -> tile: consecutive tiles per XCD (workgroups are dealt to the
  // 8 XCDs round-robin), then groups of kGroupN weight tiles, activation
  // tiles fastest inside a group
  const int nt = tiles_n * tiles_m;
  const int wg = blockIdx.x;
  const int xcd = wg & 7, kq = wg >> 3;
  const int per_x = nt >> 3, extra = nt & 7;
  const int t = xcd * per_x + (xcd < extra ? xcd : extra) + kq;
  const int grp = t / (kGroupN * tiles_m);
  const int within = t - grp * kGroupN * tiles_m;
  const int gn = tiles_n - grp * kGroupN < kGroupN ? tiles_n - grp * kGroupN : kGroupN;
  const int tn = grp * kGroupN + within % gn;
  const int tm = within / gn;
  const int64_t n0 = (int64_t)tn * BN, m0 = (int64_t)tm * BM;

  Ctx<BN, BM> c;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: keeps DMA setup scalar
  c.lane = threadIdx.x & 63;
  c.wn0 = (wave & 1) * T::WN;
  c.wm0 = (wave >> 1) * T::WM;
  c.lds0 = lds_addr(lds);
  c.S.q1 = a.steps[0];
  c.S.q2 = c.S.q1 + 2 * a.steps[1];
  c.S.Q = c.S.q2 + 2 * a.steps[2];
  c.S.t1 = a.steps[0];
  c.S.t2 = a.steps[0] + a.steps[1];

  // this wavefront's loads: wavefronts 0-1 the weight rows, 2-3 the
  // activation rows, each one half of the operand's share of a stage
  DmaConst& k = c.k;
  k.op = wave >> 1;
  k.half = wave & 1;
  k.rows_op = k.op ? BM : BN;
  const Operand& o = k.op ? a.x : a.w;
  const int64_t r0 = k.op ? m0 : n0;  // the tile's first row of the operand (below its padded rows - 31)
  k.code0 = o.q[0] + r0 * step_row_bytes(0);
  k.code1 = o.q[1] + r0 * step_row_bytes(1);
  k.code2 = o.q[2] + r0 * step_row_bytes(2);
  k.rstride0 = o.rp * step_row_bytes(0);
  k.rstride1 = o.rp * step_row_bytes(1);
  k.rstride2 = o.rp * step_row_bytes(2);
  k.last = (int)(o.rp / kRowGroup - r0 / kRowGroup - 1);
  k.op_lds = k.op ? BN / kRowGroup * 2048 : 0;
  k.op_lds6 = k.op ? BN / kRowGroup * 1536 : 0;
  // scale words (4 bytes per row and step): one half of the operand's rows,
  // 4 rows per lane; rows past the padded rows re-read the last 4
  const int per = k.rows_op / 2;
  int64_t row = k.half * per + c.lane * 4;  // row within the tile
  row = r0 + row + 4 <= o.rp ? row : o.rp - 4 - r0;
  k.soff = (uint32_t)row * kStepBlocks;
  k.sdst = (uint32_t)(T::kScaleOff + (k.op ? BN * kStepBlocks : 0) + k.half * per * kStepBlocks);
  k.smask = per / 4 >= 64 ? ~0ull : ((1ull << (per / 4)) - 1);
  k.sc = o.sc + r0 * kStepBlocks;
  k.sstride = o.rp * kStepBlocks;

  Acc<BN, BM> acc;
#pragma unroll
  for (int i = 0; i < T::TN; ++i)
#pragma unroll
    for (int j = 0; j < T::TM; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;

  // fill the ring (issues past the last stage repeat it), wait for stage 0
  DmaCursor dc;
  const int g0 = stage_group(c.S, 0);
  cursor_group(k, c.S, dc, g0, 0, c.lane);
  for (int q = 0; q < NS; ++q) {
    issue_all(k, dc, __builtin_amdgcn_readfirstlane(c.lds0 + q * T::kSlotBytes));
    cursor_next(k, c.S, dc, c.lane);
  }
  wait_vmcnt<(NS - 1) * kLoads>();
  barrier();

  // the K loop, group by group
  uint32_t st = c.lds0;
  run_group<0, FS>(c, acc, dc, st);
  run_group<1, FS>(c, acc, dc, st);
  run_group<2, FS>(c, acc, dc, st);

  // Epilogue: every load and read of the ring is done (the last stages
  // issued repeats of the last one); the bf16 tile is assembled in LDS and
  // written out as whole rows, 16 bytes per lane, so every store fills full
  // cache lines.  Lane 32 g + r, register q holds output column
  // n = 8 (q/4) + 4 g + q%4 of its fragment and output row m = r.  Rows are
  // padded by 16 bytes: the fragment writes of 32 lanes (32 rows) then fall
  // on distinct banks.
  wait_vmcnt<0>();
  wait_lgkm0();
  barrier();
  constexpr int kRowStride = BN * 2 + 16;
  static_assert(BM * kRowStride <= kLdsBytes, "epilogue tile fits LDS");
  const int r = c.lane & 31, g = c.lane >> 5;
#pragma unroll
  for (int i = 0; i < T::TN; ++i)
#pragma unroll
    for (int j = 0; j < T::TM; ++j) {
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const uint32_t lo = pack_bf16x2_rne(acc[i][j][4 * h], acc[i][j][4 * h + 1]);
        const uint32_t hi = pack_bf16x2_rne(acc[i][j][4 * h + 2], acc[i][j][4 * h + 3]);
        const uint32_t at = c.lds0 + (c.wm0 + 32 * j + r) * kRowStride + (c.wn0 + 32 * i + 8 * h + 4 * g) * 2;
        *reinterpret_cast<__attribute__((address_space(3))) u32x2*>((uintptr_t)at) = u32x2{lo, hi};
      }
      // one accumulator tile at a time: keeps the VGPR copies of the
      // accumulators few
      __builtin_amdgcn_sched_barrier(0);
    }
  __syncthreads();
  constexpr int kChunks = BN / 8;  // 16-byte chunks per row
  const int64_t M = a.x.rows, N = a.w.rows;
  for (int ch = threadIdx.x; ch < BM * kChunks; ch += kThreads) {
    const int rr = ch / kChunks, col = (ch - rr * kChunks) * 8;
    const int64_t m = m0 + rr, n = n0 + col;
    if (m >= M || n >= N) continue;
    const u32x4 v = lds_read<u32x4>(c.lds0 + rr * kRowStride + col * 2);
    uint16_t* dst = a.y + m * a.ldy + n;
    if (n + 8 <= N) {
      // streamed: the output is not read again here, and keeping it out of
      // the L2 leaves the operand panels of the tiles still running there
      __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(dst));
    } else {
      for (int e = 0; e < (int)(N - n); ++e) {
        const uint32_t wd = e < 2 ? v.x : (e < 4 ? v.y : (e < 6 ? v.z : v.w));
        dst[e] = (uint16_t)(wd >> (16 * (e & 1)));
      }
    }
  }
}

template <int BN, int BM, int FS>
static hipError_t launch_tile_fs(const GemmArgs& a, hipStream_t stream) {
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(gemm_tiled_kernel<BN, BM, FS>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBytes);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const int tn = (int)((a.w.rows + BN - 1) / BN), tm = (int)((a.x.rows + BM - 1) / BM);
  hipLaunchKernelGGL((gemm_tiled_kernel<BN, BM, FS>), dim3((unsigned)(tn * tm)), dim3(kThreads), kLdsBytes, stream, a,
                     tn, tm);
  return hipGetLastError();
}

// The format set is an instruction immediate: one kernel per set.
template <int BN, int BM>
static hipError_t launch_tile(const GemmArgs& a, hipStream_t stream) {
  switch (a.fs) {
    case 0: return launch_tile_fs<BN, BM, 0>(a, stream);
    case 1: return launch_tile_fs<BN, BM, 1>(a, stream);
    case 2: return launch_tile_fs<BN, BM, 2>(a, stream);
    case 3: return launch_tile_fs<BN, BM, 3>(a, stream);
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
  // 256 x 256 tiles when they give every CU at least one, else 256 x 128
  // (twice the tiles)
  int cus = 0;
  hipError_t e = device_cus(&cus);
  if (e != hipSuccess) return e;
  const int64_t t256 = ((a.w.rows + 255) / 256) * ((a.x.rows + 255) / 256);
  if (t256 >= cus) return launch_tile<256, 256>(a, stream);
  return launch_tile<256, 128>(a, stream);
}

}  // namespace mm
