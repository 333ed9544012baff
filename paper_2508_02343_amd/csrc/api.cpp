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

thread_local char g_err[512];

mm_status fail(mm_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int64_t round16(int64_t v) { return (v + 15) & ~(int64_t)15; }

// Checks shared by both quantise calls and the GEMM.
mm_status check_tensor(const mm_mx_tensor* t, const char* name) {
  if (!t) return fail(MM_ERR_NULL, "%s: descriptor is NULL", name);
  if (t->rows <= 0 || t->rows >= kMaxRows) return fail(MM_ERR_SHAPE, "%s: rows=%lld out of range", name, (long long)t->rows);
  if (t->K <= 0 || t->K % 32 != 0 || t->K > ((int64_t)1 << 30))
    return fail(MM_ERR_SHAPE, "%s: K=%lld must be a positive multiple of 32", name, (long long)t->K);
  const mm_split s = t->split;
  if (s.p4 < 0 || s.p6 < 0 || s.p8 < 0 || s.p4 % 32 || s.p6 % 32 || s.p8 % 32 ||
      (int64_t)s.p4 + s.p6 + s.p8 != t->K)
    return fail(MM_ERR_SPLIT, "%s: split (%d,%d,%d) must be non-negative multiples of 32 summing to K=%lld", name,
                s.p4, s.p6, s.p8, (long long)t->K);
  struct {
    const uint8_t* p;
    int64_t ld;
    int64_t need;
    const char* what;
  } bufs[4] = {{t->q4, t->ld4, (int64_t)s.p4 / 2, "q4"},
               {t->q6, t->ld6, (int64_t)s.p6 * 3 / 4, "q6"},
               {t->q8, t->ld8, (int64_t)s.p8, "q8"},
               {t->sc, t->ldsc, t->K / 32, "sc"}};
  for (auto& b : bufs) {
    if (b.need == 0) continue;
    if (!b.p) return fail(MM_ERR_NULL, "%s.%s is NULL", name, b.what);
    if (!aligned16(b.p)) return fail(MM_ERR_ALIGN, "%s.%s is not 16-byte aligned", name, b.what);
    if (b.ld % 16 != 0) return fail(MM_ERR_ALIGN, "%s.ld of %s=%lld is not a multiple of 16", name, b.what, (long long)b.ld);
    if (b.ld < round16(b.need))
      return fail(MM_ERR_SHAPE, "%s.ld of %s=%lld is below %lld", name, b.what, (long long)b.ld,
                  (long long)round16(b.need));
  }
  return MM_OK;
}

mm_status quantize(const void* x, int64_t ldx, const int32_t* perm, const mm_mx_tensor* out, void* stream,
                   const char* who) {
  g_err[0] = 0;
  if (!x) return fail(MM_ERR_NULL, "%s: input pointer is NULL", who);
  if (!perm) return fail(MM_ERR_NULL, "%s: perm is NULL", who);
  mm_status st = check_tensor(out, "out");
  if (st != MM_OK) return st;
  if (out->K > kMaxQuantK) return fail(MM_ERR_SHAPE, "%s: K=%lld exceeds %lld", who, (long long)out->K, (long long)kMaxQuantK);
  if (ldx < out->K) return fail(MM_ERR_SHAPE, "%s: ld=%lld below K=%lld", who, (long long)ldx, (long long)out->K);
  if (!aligned16(x) || ldx % 8 != 0) return fail(MM_ERR_ALIGN, "%s: input must be 16-byte aligned with ld %% 8 == 0", who);
  if (!aligned16(perm)) return fail(MM_ERR_ALIGN, "%s: perm must be 16-byte aligned", who);
  mm::QuantArgs a;
  a.x = static_cast<const uint16_t*>(x);
  a.ldx = ldx;
  a.perm = perm;
  a.rows = out->rows;
  a.K = (int)out->K;
  a.nb4 = out->split.p4 / 32;
  a.nb6 = out->split.p6 / 32;
  a.q4 = out->q4;
  a.ld4 = out->ld4;
  a.q6 = out->q6;
  a.ld6 = out->ld6;
  a.q8 = out->q8;
  a.ld8 = out->ld8;
  a.sc = out->sc;
  a.ldsc = out->ldsc;
  hipError_t e = mm::launch_quantize(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(MM_ERR_DEVICE, "%s: launch failed: %s", who, hipGetErrorString(e));
  return MM_OK;
}

mm::Operand operand(const mm_mx_tensor* t) {
  mm::Operand o;
  o.q[0] = t->q4;
  o.q[1] = t->q6;
  o.q[2] = t->q8;
  o.ld[0] = t->ld4;
  o.ld[1] = t->ld6;
  o.ld[2] = t->ld8;
  o.sc = t->sc;
  o.ldsc = t->ldsc;
  o.rows = t->rows;
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
  if (ldy < w->rows) return fail(MM_ERR_SHAPE, "mm_gemm: ldy=%lld below N=%lld", (long long)ldy, (long long)w->rows);
  if (!aligned16(y_bf16) || ldy % 8 != 0) return fail(MM_ERR_ALIGN, "mm_gemm: y must be 16-byte aligned with ldy %% 8 == 0");
  mm::GemmArgs g;
  g.w = operand(w);
  g.x = operand(a);
  g.nb[0] = a->split.p4 / 32;
  g.nb[1] = a->split.p6 / 32;
  g.nb[2] = a->split.p8 / 32;
  g.y = static_cast<uint16_t*>(y_bf16);
  g.ldy = ldy;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = a->rows <= kDirectMaxM ? mm::launch_gemm_direct(g, s) : mm::launch_gemm_tiled(g, s);
  if (e != hipSuccess) return fail(MM_ERR_DEVICE, "mm_gemm: launch failed: %s", hipGetErrorString(e));
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
  }
  return "MM_ERR_UNKNOWN";
}

const char* mm_last_error(void) { return g_err; }

int mm_abi_version(void) { return MM_ABI_VERSION; }

}  // extern "C"
