// Host side of the C ABI declared in include/micromix.h: argument validation,
// error reporting and kernel dispatch.  Nothing here allocates device memory
// or synchronises; every call only enqueues work on the caller's stream.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "../../include/micromix.h"
#include "kernels.hpp"

namespace {

constexpr int64_t kMaxQuantK = 32768;  // one row of bf16 must fit the LDS budget
constexpr int64_t kMaxRows = (int64_t)1 << 31;
// Up to this many activation rows the GEMM streams operands straight from
// global memory (memory-bound decode); above it the LDS-tiled kernel runs.
constexpr int64_t kDirectMaxM = 64;
// Calibration workspace: the workgroup maxima (nchunks * tiles <= 256 words)
// and the per-block group counts (2 * K / 256 <= 256 words), then fp64
// partial sums and means, then int32 per-slice rank counts.
constexpr int64_t kCalibHeaderBytes = 2048;

thread_local char g_err[512];

mm_status fail(mm_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Layout arithmetic of include/micromix.h.
struct Layout {
  int64_t rp;         // rows rounded up to a row group
  int nb[3];          // blocks per group
  int steps[3];       // steps per group
  int64_t bytes[4];   // q4, q6, q8, sc
};

Layout layout(int64_t rows, mm_split s) {
  Layout l;
  l.rp = (rows + mm::kRowGroup - 1) / mm::kRowGroup * mm::kRowGroup;
  const int p[3] = {s.p4, s.p6, s.p8};
  int64_t total_steps = 0;
  for (int g = 0; g < 3; ++g) {
    l.nb[g] = p[g] / 32;
    l.steps[g] = (l.nb[g] + mm::kStepBlocks - 1) / mm::kStepBlocks;
    l.bytes[g] = (int64_t)l.steps[g] * l.rp * mm::step_row_bytes(g);
    total_steps += l.steps[g];
  }
  l.bytes[3] = total_steps * l.rp * mm::kStepBlocks;
  return l;
}

mm_status check_shape(int64_t rows, int64_t K, mm_split s, const char* name) {
  if (rows <= 0 || rows >= kMaxRows) return fail(MM_ERR_SHAPE, "%s: rows=%lld out of range", name, (long long)rows);
  if (K <= 0 || K % 32 != 0 || K > ((int64_t)1 << 30))
    return fail(MM_ERR_SHAPE, "%s: K=%lld must be a positive multiple of 32", name, (long long)K);
  if (s.p4 < 0 || s.p6 < 0 || s.p8 < 0 || s.p4 % 32 || s.p6 % 32 || s.p8 % 32 || (int64_t)s.p4 + s.p6 + s.p8 != K)
    return fail(MM_ERR_SPLIT, "%s: split (%d,%d,%d) must be non-negative multiples of 32 summing to K=%lld", name,
                s.p4, s.p6, s.p8, (long long)K);
  return MM_OK;
}

// Format set of a descriptor (the kernels' fs): bit 0 E2M3, bit 1 E5M2.
int format_set(const mm_mx_tensor* t) { return (t->formats.fp6 == MM_FP6_E2M3 ? 1 : 0) | (t->formats.fp8 == MM_FP8_E5M2 ? 2 : 0); }

// Checks shared by both quantise calls and the GEMM.
mm_status check_tensor(const mm_mx_tensor* t, const char* name) {
  if (!t) return fail(MM_ERR_NULL, "%s: descriptor is NULL", name);
  mm_status st = check_shape(t->rows, t->K, t->split, name);
  if (st != MM_OK) return st;
  if ((t->formats.fp6 != MM_FP6_E3M2 && t->formats.fp6 != MM_FP6_E2M3) ||
      (t->formats.fp8 != MM_FP8_E4M3 && t->formats.fp8 != MM_FP8_E5M2))
    return fail(MM_ERR_FORMAT, "%s: unknown element format (fp6=%d, fp8=%d)", name, t->formats.fp6, t->formats.fp8);
  const Layout l = layout(t->rows, t->split);
  const uint8_t* ptrs[4] = {t->q4, t->q6, t->q8, t->sc};
  const char* what[4] = {"q4", "q6", "q8", "sc"};
  for (int b = 0; b < 4; ++b) {
    if (l.bytes[b] == 0) continue;
    if (!ptrs[b]) return fail(MM_ERR_NULL, "%s.%s is NULL", name, what[b]);
    if (!aligned16(ptrs[b])) return fail(MM_ERR_ALIGN, "%s.%s is not 16-byte aligned", name, what[b]);
  }
  return MM_OK;
}

mm_status quantize(const void* x, int64_t ldx, const int32_t* perm, const mm_mx_tensor* out, void* stream,
                   const char* who, const void* gamma = nullptr, float eps = 0.0f) {
  g_err[0] = 0;
  if (!x) return fail(MM_ERR_NULL, "%s: input pointer is NULL", who);
  if (!perm) return fail(MM_ERR_NULL, "%s: perm is NULL", who);
  const bool norm = gamma != nullptr;
  mm_status st = check_tensor(out, "out");
  if (st != MM_OK) return st;
  if (out->K > kMaxQuantK) return fail(MM_ERR_SHAPE, "%s: K=%lld exceeds %lld", who, (long long)out->K, (long long)kMaxQuantK);
  if (ldx < out->K) return fail(MM_ERR_SHAPE, "%s: ld=%lld below K=%lld", who, (long long)ldx, (long long)out->K);
  if (!aligned16(x) || ldx % 8 != 0) return fail(MM_ERR_ALIGN, "%s: input must be 16-byte aligned with ld %% 8 == 0", who);
  if (!aligned16(perm)) return fail(MM_ERR_ALIGN, "%s: perm must be 16-byte aligned", who);
  if (norm && !(eps > 0.0f && eps <= 3.0e38f))
    return fail(MM_ERR_VALUE, "%s: eps=%g must be finite and positive", who, (double)eps);
  if (norm && !aligned16(gamma)) return fail(MM_ERR_ALIGN, "%s: gamma must be 16-byte aligned", who);
  const Layout l = layout(out->rows, out->split);
  mm::QuantArgs a;
  a.x = static_cast<const uint16_t*>(x);
  a.ldx = ldx;
  a.perm = perm;
  a.rows = out->rows;
  a.rp = l.rp;
  a.K = (int)out->K;
  for (int g = 0; g < 3; ++g) {
    a.nb[g] = l.nb[g];
    a.steps[g] = l.steps[g];
  }
  a.q[0] = out->q4;
  a.q[1] = out->q6;
  a.q[2] = out->q8;
  a.sc = out->sc;
  a.fs = format_set(out);
  a.norm = norm ? 1 : 0;
  a.gamma = static_cast<const uint16_t*>(gamma);
  a.eps = eps;
  hipError_t e = mm::launch_quantize(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(MM_ERR_DEVICE, "%s: launch failed: %s", who, hipGetErrorString(e));
  return MM_OK;
}

// Row chunks of the calibration column sums: at most one workgroup per CU
// over the 512-channel tiles (more concurrent row streams lose DRAM
// locality), 1 .. 128 chunks, at least 64 rows per chunk.  Depends only on
// (rows, K), so results are reproducible.
struct CalibPlan {
  int nchunks;
  int tiles;
  int64_t chunk_rows;
  int64_t bytes;  // workspace
};

CalibPlan calib_plan(int64_t rows, int64_t K) {
  CalibPlan p;
  p.tiles = (int)((K + 511) / 512);
  int64_t n = mm::kCalibMaxWorkgroups / p.tiles;
  n = n < 1 ? 1 : (n > 128 ? 128 : n);
  const int64_t max_n = (rows + 63) / 64;
  if (n > max_n) n = max_n;
  p.chunk_rows = (rows + n - 1) / n;
  p.nchunks = (int)((rows + p.chunk_rows - 1) / p.chunk_rows);
  const int64_t nslices = (K + mm::kCalibSlice - 1) / mm::kCalibSlice;
  p.bytes = kCalibHeaderBytes + ((int64_t)p.nchunks + 1) * K * (int64_t)sizeof(double) +
            nslices * K * (int64_t)sizeof(int32_t);
  return p;
}

mm_status check_calib_shape(int64_t rows, int64_t K, const char* who) {
  if (rows <= 0 || rows >= kMaxRows) return fail(MM_ERR_SHAPE, "%s: rows=%lld out of range", who, (long long)rows);
  if (K <= 0 || K % 32 != 0 || K > kMaxQuantK)
    return fail(MM_ERR_SHAPE, "%s: K=%lld must be a positive multiple of 32, at most %lld", who, (long long)K,
                (long long)kMaxQuantK);
  return MM_OK;
}

mm::Operand operand(const mm_mx_tensor* t) {
  mm::Operand o;
  o.q[0] = t->q4;
  o.q[1] = t->q6;
  o.q[2] = t->q8;
  o.sc = t->sc;
  o.rows = t->rows;
  o.rp = layout(t->rows, t->split).rp;
  return o;
}

}  // namespace

extern "C" {

mm_status mm_quantize_act(const void* x_bf16, int64_t ldx, const int32_t* perm, const mm_mx_tensor* out,
                          void* stream) {
  return quantize(x_bf16, ldx, perm, out, stream, "mm_quantize_act");
}

mm_status mm_quantize_weight(const void* w_bf16, int64_t ldw, const int32_t* perm, const mm_mx_tensor* out,
                             void* stream) {
  return quantize(w_bf16, ldw, perm, out, stream, "mm_quantize_weight");
}

mm_status mm_rmsnorm_quantize_act(const void* x_bf16, int64_t ldx, const void* gamma_bf16, float eps,
                                  const int32_t* perm, const mm_mx_tensor* out, void* stream) {
  if (!gamma_bf16) {
    g_err[0] = 0;
    return fail(MM_ERR_NULL, "mm_rmsnorm_quantize_act: gamma is NULL");
  }
  return quantize(x_bf16, ldx, perm, out, stream, "mm_rmsnorm_quantize_act", gamma_bf16, eps);
}

mm_status mm_gemm(const mm_mx_tensor* a, const mm_mx_tensor* w, void* y_bf16, int64_t ldy, void* stream) {
  g_err[0] = 0;
  mm_status st = check_tensor(a, "a");
  if (st != MM_OK) return st;
  st = check_tensor(w, "w");
  if (st != MM_OK) return st;
  if (!y_bf16) return fail(MM_ERR_NULL, "mm_gemm: y is NULL");
  if (a->K != w->K) return fail(MM_ERR_SHAPE, "mm_gemm: K differs (%lld vs %lld)", (long long)a->K, (long long)w->K);
  if (a->split.p4 != w->split.p4 || a->split.p6 != w->split.p6 || a->split.p8 != w->split.p8)
    return fail(MM_ERR_SHAPE, "mm_gemm: a and w must share the split");
  if (format_set(a) != format_set(w)) return fail(MM_ERR_FORMAT, "mm_gemm: a and w must share the element formats");
  if (ldy < w->rows) return fail(MM_ERR_SHAPE, "mm_gemm: ldy=%lld below N=%lld", (long long)ldy, (long long)w->rows);
  if (!aligned16(y_bf16) || ldy % 8 != 0) return fail(MM_ERR_ALIGN, "mm_gemm: y must be 16-byte aligned with ldy %% 8 == 0");
  mm::GemmArgs g;
  g.w = operand(w);
  g.x = operand(a);
  const Layout l = layout(a->rows, a->split);
  for (int k = 0; k < 3; ++k) g.steps[k] = l.steps[k];
  g.y = static_cast<uint16_t*>(y_bf16);
  g.ldy = ldy;
  g.fs = format_set(a);
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = a->rows <= kDirectMaxM ? mm::launch_gemm_direct(g, s) : mm::launch_gemm_tiled(g, s);
  if (e != hipSuccess) return fail(MM_ERR_DEVICE, "mm_gemm: launch failed: %s", hipGetErrorString(e));
  return MM_OK;
}

mm_status mm_calibrate_workspace_size(int64_t rows, int64_t K, int64_t* bytes) {
  g_err[0] = 0;
  if (!bytes) return fail(MM_ERR_NULL, "mm_calibrate_workspace_size: bytes is NULL");
  mm_status st = check_calib_shape(rows, K, "mm_calibrate_workspace_size");
  if (st != MM_OK) return st;
  *bytes = calib_plan(rows, K).bytes;
  return MM_OK;
}

namespace {

// mm_calibrate and mm_calibrate_no_alloc: workspace == nullptr takes the
// library's static scratch (looked up, never allocated).
mm_status calibrate(const void* x_bf16, int64_t rows, int64_t K, int64_t ldx, mm_formats formats, void* workspace,
                    int64_t workspace_bytes, int32_t* perm_out, int32_t* split_out, void* stream, const char* who) {
  const bool own = workspace == nullptr;
  if (!x_bf16 || !perm_out || !split_out) return fail(MM_ERR_NULL, "%s: a pointer is NULL", who);
  mm_status st = check_calib_shape(rows, K, who);
  if (st != MM_OK) return st;
  if (ldx < K) return fail(MM_ERR_SHAPE, "%s: ld=%lld below K=%lld", who, (long long)ldx, (long long)K);
  if ((formats.fp6 != MM_FP6_E3M2 && formats.fp6 != MM_FP6_E2M3) ||
      (formats.fp8 != MM_FP8_E4M3 && formats.fp8 != MM_FP8_E5M2))
    return fail(MM_ERR_FORMAT, "%s: unknown element format (fp6=%d, fp8=%d)", who, formats.fp6, formats.fp8);
  const CalibPlan p = calib_plan(rows, K);
  if ((int64_t)p.nchunks * p.tiles * 4 > kCalibHeaderBytes / 2 || 2 * ((K + 255) / 256) * 4 > kCalibHeaderBytes / 2)
    return fail(MM_ERR_SHAPE, "%s: internal plan exceeds the workspace header", who);
  if (own && p.bytes > mm::kCalibScratchBytes)
    return fail(MM_ERR_WORKSPACE, "%s: rows=%lld, K=%lld need %lld bytes of workspace, beyond the %lld-byte static "
                "scratch; call mm_calibrate with a workspace instead", who, (long long)rows, (long long)K,
                (long long)p.bytes, (long long)mm::kCalibScratchBytes);
  if (!own && workspace_bytes < p.bytes)
    return fail(MM_ERR_WORKSPACE, "%s: workspace of %lld bytes, %lld needed", who, (long long)workspace_bytes,
                (long long)p.bytes);
  if (!aligned16(x_bf16) || ldx % 8 != 0) return fail(MM_ERR_ALIGN, "%s: input must be 16-byte aligned with ld %% 8 == 0", who);
  if ((!own && !aligned16(workspace)) || !aligned16(perm_out) || ((uintptr_t)split_out & 3u))
    return fail(MM_ERR_ALIGN, "%s: workspace and perm must be 16-byte aligned, split 4-byte aligned", who);
  if (own) {
    hipError_t e = mm::calibrate_scratch(&workspace);
    if (e != hipSuccess) return fail(MM_ERR_DEVICE, "%s: static scratch lookup failed: %s", who, hipGetErrorString(e));
  }
  mm::CalibArgs a;
  a.x = static_cast<const uint16_t*>(x_bf16);
  a.ldx = ldx;
  a.rows = rows;
  a.K = (int)K;
  a.nchunks = p.nchunks;
  a.chunk_rows = p.chunk_rows;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  a.wgmax = reinterpret_cast<uint32_t*>(ws);
  a.nmax = p.nchunks * p.tiles;
  a.counts = reinterpret_cast<int32_t*>(ws + kCalibHeaderBytes / 2);
  a.partial = reinterpret_cast<double*>(ws + kCalibHeaderBytes);
  a.mean = a.partial + (int64_t)p.nchunks * K;
  a.slice_counts = reinterpret_cast<int32_t*>(a.mean + K);
  a.perm = perm_out;
  a.split = split_out;
  a.fp6_e2m3 = formats.fp6 == MM_FP6_E2M3;
  hipError_t e = mm::launch_calibrate(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(MM_ERR_DEVICE, "%s: launch failed: %s", who, hipGetErrorString(e));
  return MM_OK;
}

}  // namespace

mm_status mm_calibrate(const void* x_bf16, int64_t rows, int64_t K, int64_t ldx, mm_formats formats, void* workspace,
                       int64_t workspace_bytes, int32_t* perm_out, int32_t* split_out, void* stream) {
  g_err[0] = 0;
  if (!workspace) return fail(MM_ERR_NULL, "mm_calibrate: a pointer is NULL");
  return calibrate(x_bf16, rows, K, ldx, formats, workspace, workspace_bytes, perm_out, split_out, stream,
                   "mm_calibrate");
}

mm_status mm_calibrate_no_alloc(const void* x_bf16, int64_t rows, int64_t K, int64_t ldx, mm_formats formats,
                                int32_t* perm_out, int32_t* split_out, void* stream) {
  g_err[0] = 0;
  return calibrate(x_bf16, rows, K, ldx, formats, nullptr, 0, perm_out, split_out, stream, "mm_calibrate_no_alloc");
}

mm_status mm_mx_layout_sizes(int64_t rows, int64_t K, mm_split split, mm_mx_sizes* out) {
  g_err[0] = 0;
  if (!out) return fail(MM_ERR_NULL, "mm_mx_layout_sizes: out is NULL");
  mm_status st = check_shape(rows, K, split, "mm_mx_layout_sizes");
  if (st != MM_OK) return st;
  const Layout l = layout(rows, split);
  out->q4 = l.bytes[0];
  out->q6 = l.bytes[1];
  out->q8 = l.bytes[2];
  out->sc = l.bytes[3];
  return MM_OK;
}

const char* mm_status_str(mm_status s) {
  switch (s) {
    case MM_OK: return "MM_OK";
    case MM_ERR_NULL: return "MM_ERR_NULL";
    case MM_ERR_SHAPE: return "MM_ERR_SHAPE";
    case MM_ERR_SPLIT: return "MM_ERR_SPLIT";
    case MM_ERR_ALIGN: return "MM_ERR_ALIGN";
    case MM_ERR_FORMAT: return "MM_ERR_FORMAT";
    case MM_ERR_DEVICE: return "MM_ERR_DEVICE";
    case MM_ERR_WORKSPACE: return "MM_ERR_WORKSPACE";
    case MM_ERR_VALUE: return "MM_ERR_VALUE";
  }
  return "MM_ERR_UNKNOWN";
}

const char* mm_last_error(void) { return g_err; }

int mm_abi_version(void) { return MM_ABI_VERSION; }

}  // extern "C"
