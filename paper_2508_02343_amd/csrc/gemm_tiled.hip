// Mixed MX GEMM for prefill shapes (many activation rows): compute-bound, so
// operand tiles are staged through LDS and reused across the workgroup.
//
// Workgroup tile: 128 weight rows (output columns n) x 128 activation rows
// (output rows m); four wavefronts in a 2 x 2 grid, each owning a 64 x 64
// output sub-tile = 4 x 4 MFMA tiles of 16 x 16 in fp32 registers.  The K
// loop visits the E2M1 group, then E3M2, then E4M3 (Sec. 3.1 group order),
// 128 channels (4 MX blocks) per step, all accumulating into the same
// registers (Sec. 3.2 "GEMM kernel": one fp32 accumulation, bf16 result).
//
// Per step, global -> registers -> LDS double buffering: the loads of step
// s+1 are in flight while step s is multiplied from the other LDS buffer.
// LDS rows are padded (80 / 112 / 144 bytes for 64 / 96 / 128 data bytes)
// so that a wavefront's 16-byte fragment reads spread over all banks.
#include "gemm_common.hpp"

namespace mm {

namespace tiled {

constexpr int BN = 128;  // weight rows per workgroup
constexpr int BM = 128;  // activation rows per workgroup
constexpr int kThreads = 256;

__host__ __device__ constexpr int row_bytes(int G) { return G == 0 ? 64 : (G == 1 ? 96 : 128); }
__host__ __device__ constexpr int lds_stride(int G) { return G == 0 ? 80 : (G == 1 ? 112 : 144); }
__host__ __device__ constexpr int chunks_per_row(int G) { return row_bytes(G) / 16; }

constexpr int kOpBytes = 128 * 144;                 // one operand tile, largest stride
constexpr int kStageBytes = 2 * kOpBytes + 2 * 128 * 4;  // both operands + their scales
constexpr int kLdsBytes = 2 * kStageBytes;

struct Stage {
  uint8_t* op[2];  // 0 = weight tile, 1 = activation tile
  uint8_t* sc[2];  // [128 rows][4 blocks] E8M0 bytes per operand
};

__device__ __forceinline__ Stage stage_ptrs(uint8_t* lds, int s) {
  Stage st;
  uint8_t* base = lds + s * kStageBytes;
  st.op[0] = base;
  st.op[1] = base + kOpBytes;
  st.sc[0] = base + 2 * kOpBytes;
  st.sc[1] = base + 2 * kOpBytes + 512;
  return st;
}

// Registers holding one step's global loads until they are written to LDS.
struct Staging {
  uint4 v[8];
  uint32_t sc[4];  // raw scale bytes; packed only when written to LDS, so
                   // that nothing waits for the loads before the MFMAs run
};

// Operand pointers of one group, copied out of the kernel arguments (taking
// the address of the argument block would force it into scratch memory).
struct Ctx {
  const uint8_t* q[2];  // weight / activation codes of the current group
  int64_t ld[2];
  const uint8_t* sc[2];
  int64_t ldsc[2];
  int64_t row0[2];  // first weight row / activation row of this workgroup
  int64_t rows[2];
  int gblk0;        // first block of the group inside a scale row
};

template <int G>
__device__ __forceinline__ Ctx make_ctx(const GemmArgs& a) {
  Ctx c;
  c.q[0] = a.w.q[G];
  c.q[1] = a.x.q[G];
  c.ld[0] = a.w.ld[G];
  c.ld[1] = a.x.ld[G];
  c.sc[0] = a.w.sc;
  c.sc[1] = a.x.sc;
  c.ldsc[0] = a.w.ldsc;
  c.ldsc[1] = a.x.ldsc;
  c.row0[0] = (int64_t)blockIdx.x * BN;
  c.row0[1] = (int64_t)blockIdx.y * BM;
  c.rows[0] = a.w.rows;
  c.rows[1] = a.x.rows;
  c.gblk0 = G == 0 ? 0 : (G == 1 ? a.nb[0] : a.nb[0] + a.nb[1]);
  return c;
}

template <int G>
__device__ __forceinline__ void load_step(const Ctx& c, int blk0, int nvalid, Staging& s) {
  constexpr int CPR = chunks_per_row(G);
  constexpr int BB = block_bytes(G);
  const int tid = threadIdx.x;
  const int valid_bytes = nvalid * BB;
#pragma unroll
  for (int k = 0; k < CPR; ++k) {
    // chunk id q = 256 k + tid over both operands; 128 * CPR = 256 * (CPR / 2)
    // chunks per operand, so the operand index is known at compile time
    const int op = k / (CPR / 2);
    const int rem = kThreads * (k % (CPR / 2)) + tid;
    const int r = rem / CPR;
    const int ch = rem - r * CPR;
    int64_t row = c.row0[op] + r;
    row = row < c.rows[op] ? row : c.rows[op] - 1;
    const uint8_t* src = c.q[op] + row * c.ld[op] + blk0 * BB + ch * 16;
    uint4 v = gload16(ch * 16 < valid_bytes ? src : kZeroCodes);
    if constexpr (G == 1) {
      // an E3M2 block (24 bytes) can end in the middle of a chunk: clear the
      // bytes past the group's end so that LDS holds zero codes there
      const bool half = ch * 16 + 8 == valid_bytes;
      v.z = half ? 0u : v.z;
      v.w = half ? 0u : v.w;
    }
    s.v[k] = v;
  }
  // scales: thread t loads the 4 bytes of (operand t / 128, row t % 128)
  {
    // (selects, not array indexing: a lane-dependent index would put the
    // context in scratch memory)
    const bool op = tid >= 128;
    const int r = tid & 127;
    const int64_t nrows = op ? c.rows[1] : c.rows[0];
    int64_t row = (op ? c.row0[1] : c.row0[0]) + r;
    row = row < nrows ? row : nrows - 1;
    const uint8_t* p = (op ? c.sc[1] : c.sc[0]) + row * (op ? c.ldsc[1] : c.ldsc[0]) + c.gblk0 + blk0;
#pragma unroll
    for (int j = 0; j < 4; ++j) s.sc[j] = (uint32_t)load_scale(p, j, j < nvalid);
  }
}

template <int G>
__device__ __forceinline__ void store_step(const Stage& st, const Staging& s) {
  constexpr int CPR = chunks_per_row(G);
  constexpr int STR = lds_stride(G);
  const int tid = threadIdx.x;
#pragma unroll
  for (int k = 0; k < CPR; ++k) {
    const int op = k / (CPR / 2);
    const int rem = kThreads * (k % (CPR / 2)) + tid;
    const int r = rem / CPR;
    const int ch = rem - r * CPR;
    *reinterpret_cast<uint4*>(st.op[op] + r * STR + ch * 16) = s.v[k];
  }
  const uint32_t w = s.sc[0] | (s.sc[1] << 8) | (s.sc[2] << 16) | (s.sc[3] << 24);
  *reinterpret_cast<uint32_t*>((tid >= 128 ? st.sc[1] : st.sc[0]) + (tid & 127) * 4) = w;
}

// One lane's fragment (row `row`, block g of the step) of a staged operand
// tile.  Bytes of blocks past the group's end were stored as zeros, and their
// scales as 1.0, so no masking is needed here.
template <int G>
__device__ __forceinline__ v8i read_frag(const uint8_t* op, int row, int g) {
  constexpr int STR = lds_stride(G);
  v8i v;
  const uint8_t* p = op + row * STR;
  if constexpr (G == 0) {
    const uint4 d = *reinterpret_cast<const uint4*>(p + 16 * g);
    v[0] = (int)d.x;
    v[1] = (int)d.y;
    v[2] = (int)d.z;
    v[3] = (int)d.w;
    v[4] = v[5] = v[6] = v[7] = 0;
  } else if constexpr (G == 1) {
    const uint2* s = reinterpret_cast<const uint2*>(p + 24 * g);
    const uint2 d0 = s[0], d1 = s[1], d2 = s[2];
    v[0] = (int)d0.x;
    v[1] = (int)d0.y;
    v[2] = (int)d1.x;
    v[3] = (int)d1.y;
    v[4] = (int)d2.x;
    v[5] = (int)d2.y;
    v[6] = v[7] = 0;
  } else {
    const uint4 lo = *reinterpret_cast<const uint4*>(p + 16 * g);
    const uint4 hi = *reinterpret_cast<const uint4*>(p + 64 + 16 * g);
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

template <int G>
__device__ __forceinline__ void compute_step(const Stage& st, int wn0, int wm0, v4f (&acc)[4][4]) {
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, r = lane & 15;
  v8i wf[4], xf[4];
  int ws[4], xs[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = wn0 + 16 * i + r;
    wf[i] = read_frag<G>(st.op[0], row, g);
    ws[i] = st.sc[0][row * 4 + g];
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int row = wm0 + 16 * j + r;
    xf[j] = read_frag<G>(st.op[1], row, g);
    xs[j] = st.sc[1][row * 4 + g];
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) MM_MFMA_GROUP(G, acc[i][j], wf[i], xf[j], ws[i], xs[j]);
}

// All K steps of one group, double-buffered through LDS.  `stage` is the LDS
// buffer the group starts in; it is left pointing at the next free buffer.
template <int G>
__device__ __forceinline__ void run_group(const GemmArgs& a, uint8_t* lds, int& stage, int wn0, int wm0,
                                          v4f (&acc)[4][4]) {
  const int nb = a.nb[G];
  if (nb == 0) return;
  const int S = (nb + 3) >> 2;
  const Ctx c = make_ctx<G>(a);
  Staging stg;
  load_step<G>(c, 0, nb < 4 ? nb : 4, stg);
  store_step<G>(stage_ptrs(lds, stage), stg);
  __syncthreads();
  // steady state: no branches inside, so the scheduler keeps the order
  // global loads (step ks+1) -> MFMAs (step ks) -> LDS writes (step ks+1)
  for (int ks = 0; ks + 1 < S; ++ks) {
    const int left = nb - 4 * (ks + 1);
    load_step<G>(c, 4 * (ks + 1), left < 4 ? left : 4, stg);
    compute_step<G>(stage_ptrs(lds, stage), wn0, wm0, acc);
    // keep the LDS writes (which wait for the global loads) behind the
    // MFMAs, so the loads' latency overlaps the matrix work
    __builtin_amdgcn_sched_barrier(0);
    store_step<G>(stage_ptrs(lds, stage ^ 1), stg);
    __syncthreads();
    stage ^= 1;
  }
  compute_step<G>(stage_ptrs(lds, stage), wn0, wm0, acc);
  __syncthreads();
  stage ^= 1;
}

}  // namespace tiled

using namespace tiled;

__global__ __launch_bounds__(kThreads) void gemm_tiled_kernel(GemmArgs a) {
  extern __shared__ __align__(16) uint8_t lds[];
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int wn0 = (wave & 1) * 64;   // wave's weight-row offset in the tile
  const int wm0 = (wave >> 1) * 64;  // wave's activation-row offset
  const int64_t n_base = (int64_t)blockIdx.x * BN;
  const int64_t m_base = (int64_t)blockIdx.y * BM;

  v4f acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  int stage = 0;
  run_group<0>(a, lds, stage, wn0, wm0, acc);
  run_group<1>(a, lds, stage, wn0, wm0, acc);
  run_group<2>(a, lds, stage, wn0, wm0, acc);

  const int lane = tid & 63;
  const int g = lane >> 4, r = lane & 15;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      store_out4(a, m_base + wm0 + 16 * j + r, n_base + wn0 + 16 * i + 4 * g, acc[i][j], a.x.rows, a.w.rows);
}

hipError_t launch_gemm_tiled(const GemmArgs& a, hipStream_t stream) {
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(gemm_tiled_kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBytes);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const dim3 grid((unsigned)((a.w.rows + BN - 1) / BN), (unsigned)((a.x.rows + BM - 1) / BM));
  hipLaunchKernelGGL(gemm_tiled_kernel, grid, dim3(kThreads), kLdsBytes, stream, a);
  return hipGetLastError();
}

}  // namespace mm
