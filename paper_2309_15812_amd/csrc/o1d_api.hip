// C ABI of the oriented 1D depthwise convolution library (declared in
// include/o1d.h): argument validation, status codes, per-thread error text
// and dispatch to the kernel launchers.  No device memory is allocated here.
#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "o1d.h"
#include "o1d_launch.h"
#include "o1d_plan.h"
#include "o1d_line.h"
#include "o1d_strip.h"

namespace {

thread_local char g_last_error[512] = "";

o1d_status_t fail(o1d_status_t st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return st;
}

o1d_status_t ok() {
  g_last_error[0] = '\0';
  return O1D_OK;
}

size_t elem_size(o1d_dtype_t dt) { return dt == O1D_BF16 ? 2u : 4u; }

bool overlaps(const void* a, size_t abytes, const void* b, size_t bbytes) {
  const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + bbytes && b0 < a0 + abytes;
}

// Checks shared by all entry points.  Sets *empty when there is nothing to
// compute over the batch/plane (N, H or W zero) or no channel (C zero).
o1d_status_t check_sizes(const char* fn, int N, int C, int H, int W, int K, o1d_dtype_t dt) {
  if (dt != O1D_F32 && dt != O1D_BF16) return fail(O1D_ERR_INVALID, "%s: unknown dtype %d", fn, (int)dt);
  if (N < 0 || C < 0 || H < 0 || W < 0)
    return fail(O1D_ERR_INVALID, "%s: negative size N=%d C=%d H=%d W=%d", fn, N, C, H, W);
  if (K < 1 || (K % 2) == 0)
    return fail(O1D_ERR_INVALID, "%s: K=%d must be odd and positive (pad = K/2 centres the kernel)", fn, K);
  if (K > O1D_MAX_K) return fail(O1D_ERR_UNSUPPORTED, "%s: K=%d exceeds O1D_MAX_K=%d", fn, K, O1D_MAX_K);
  if (C > 65535 || N > 65535)
    return fail(O1D_ERR_UNSUPPORTED, "%s: N=%d or C=%d exceeds the 65535 grid limit", fn, N, C);
  if ((long long)H * (long long)W > (1ll << 30))
    return fail(O1D_ERR_UNSUPPORTED, "%s: plane %dx%d exceeds 2^30 elements", fn, H, W);
  return O1D_OK;
}

// Kernel family: the line kernels cover K <= 63, planes up to 64 columns and
// haloed tiles that fit in LDS; everything else takes the general tiled
// kernels.  O1D_KERNEL=tiled forces the tiled kernels (a comparison aid).
bool line_allowed() {
  const char* e = getenv("O1D_KERNEL");
  return !(e && e[0] == 't');
}

o1d::line::LinePlan line_plan(int N, int C, int H, int W, int K, int sign, int kind, bool vec_ok) {
  if (!line_allowed()) return o1d::line::LinePlan();
  return o1d::line::plan_line(N, C, H, W, K, sign, kind, vec_ok);
}

// Vector staging needs 16-byte (float32) or 8-byte (bfloat16) aligned tensors.
bool vec_aligned(const void* p, o1d_dtype_t dt) { return ((uintptr_t)p % (dt == O1D_BF16 ? 8u : 16u)) == 0; }

// The workspace size must not depend on pointer alignment: take the larger
// partial count of the kernels that aligned and unaligned tensors select
// (the line kernels need aligned tensors; otherwise the tiled kernels run).
o1d::strip::Plan strip_wgrad_plan(int N, int C, int H, int W, int K, bool vec_ok) {
  if (!line_allowed()) return o1d::strip::Plan();
  return o1d::strip::plan_strip(N, C, H, W, K, 1, 1, vec_ok);
}

size_t wgrad_workspace(int N, int C, int H, int W, int K) {
  const o1d::strip::Plan sa = strip_wgrad_plan(N, C, H, W, K, true);
  if (sa.ok) {
    // aligned tensors take the strip kernel, unaligned ones a line or tiled kernel
    const o1d::line::LinePlan b = line_plan(N, C, H, W, K, 1, 1, false);
    const size_t pb = b.ok ? (size_t)b.blocks_n : o1d::plan_wgrad(N, C, H, W, K).parts();
    const size_t parts = (size_t)sa.blocks_n > pb ? (size_t)sa.blocks_n : pb;
    return parts * (size_t)C * (size_t)K * sizeof(float);
  }
  const o1d::line::LinePlan a = line_plan(N, C, H, W, K, 1, 1, true);
  const o1d::line::LinePlan b = line_plan(N, C, H, W, K, 1, 1, false);
  const size_t tiled = o1d::plan_wgrad(N, C, H, W, K).parts();
  const size_t pa = a.ok ? (size_t)a.blocks_n : tiled, pb = b.ok ? (size_t)b.blocks_n : tiled;
  const size_t parts = pa > pb ? pa : pb;
  return parts * (size_t)C * (size_t)K * sizeof(float);
}

o1d_status_t hip_status(const char* fn, hipError_t e) {
  if (e != hipSuccess) return fail(O1D_ERR_HIP, "%s: kernel launch failed: %s", fn, hipGetErrorString(e));
  return ok();
}

o1d_status_t gather_entry(const char* fn, const void* in, const void* w, const float* theta, void* out, int N, int C,
                          int H, int W, int K, o1d_dtype_t dt, void* stream, int sign) {
  o1d_status_t st = check_sizes(fn, N, C, H, W, K, dt);
  if (st != O1D_OK) return st;
  const size_t elems = (size_t)N * C * H * W;
  if (elems == 0) return ok();
  if (!in || !w || !theta || !out) return fail(O1D_ERR_INVALID, "%s: NULL tensor pointer", fn);
  const size_t bytes = elems * elem_size(dt);
  if (overlaps(in, bytes, out, bytes)) return fail(O1D_ERR_INVALID, "%s: output overlaps input", fn);
  (void)hipGetLastError();
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool va = vec_aligned(in, dt) && vec_aligned(out, dt);
  if (line_allowed()) {
    const o1d::strip::Plan sp = o1d::strip::plan_strip(N, C, H, W, K, sign, 0, va);
    if (sp.ok) return hip_status(fn, o1d::launch_gather_strip((o1d::Dtype)dt, sp, in, w, theta, out, s));
  }
  const o1d::line::LinePlan lp = line_plan(N, C, H, W, K, sign, 0, va);
  if (lp.ok) return hip_status(fn, o1d::launch_gather_line((o1d::Dtype)dt, lp, in, w, theta, out, s));
  return hip_status(fn, o1d::launch_gather((o1d::Dtype)dt, in, w, theta, out, N, C, H, W, K, sign, s));
}

// Weight gradient after validation: the strip kernel, else a line kernel,
// else the tiled kernels (the workspace covers all three, see above).
o1d_status_t wgrad_dispatch(const char* fn, const void* x, const void* dy, const float* theta, void* dw, int N, int C,
                            int H, int W, int K, o1d_dtype_t dt, void* workspace, hipStream_t s) {
  const bool va = vec_aligned(x, dt) && vec_aligned(dy, dt);
  const o1d::strip::Plan sp = strip_wgrad_plan(N, C, H, W, K, va);
  if (sp.ok)
    return hip_status(fn, o1d::launch_wgrad_strip((o1d::Dtype)dt, sp, x, dy, theta, dw,
                                                  static_cast<float*>(workspace), s));
  const o1d::line::LinePlan lp = line_plan(N, C, H, W, K, 1, 1, va);
  if (lp.ok)
    return hip_status(fn, o1d::launch_wgrad_line((o1d::Dtype)dt, lp, x, dy, theta, dw,
                                                 static_cast<float*>(workspace), s));
  return hip_status(fn, o1d::launch_wgrad((o1d::Dtype)dt, x, dy, theta, dw, static_cast<float*>(workspace), N, C, H,
                                          W, K, s));
}

}  // namespace

extern "C" {

size_t o1d_bwd_weight_workspace_bytes(int N, int C, int H, int W, int K, o1d_dtype_t dtype) {
  if (check_sizes("o1d_bwd_weight_workspace_bytes", N, C, H, W, K, dtype) != O1D_OK) return 0;
  if ((size_t)N * C * H * W == 0) return 0;
  return wgrad_workspace(N, C, H, W, K);
}

o1d_status_t o1d_fwd(const void* x, const void* w, const float* theta_deg, void* y, int N, int C, int H, int W, int K,
                     o1d_dtype_t dtype, void* stream) {
  return gather_entry("o1d_fwd", x, w, theta_deg, y, N, C, H, W, K, dtype, stream, +1);
}

o1d_status_t o1d_bwd_input(const void* dy, const void* w, const float* theta_deg, void* dx, int N, int C, int H,
                           int W, int K, o1d_dtype_t dtype, void* stream) {
  return gather_entry("o1d_bwd_input", dy, w, theta_deg, dx, N, C, H, W, K, dtype, stream, -1);
}

o1d_status_t o1d_bwd_weight(const void* x, const void* dy, const float* theta_deg, void* dw, int N, int C, int H,
                            int W, int K, o1d_dtype_t dtype, void* workspace, size_t workspace_bytes, void* stream) {
  const char* fn = "o1d_bwd_weight";
  o1d_status_t st = check_sizes(fn, N, C, H, W, K, dtype);
  if (st != O1D_OK) return st;
  if (C == 0) return ok();
  if (!dw) return fail(O1D_ERR_INVALID, "%s: NULL dw pointer", fn);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t elems = (size_t)N * C * H * W;
  (void)hipGetLastError();
  if (elems == 0) return hip_status(fn, o1d::launch_zero((o1d::Dtype)dtype, dw, (size_t)C * K, s));
  if (!x || !dy || !theta_deg) return fail(O1D_ERR_INVALID, "%s: NULL tensor pointer", fn);
  const size_t need = o1d_bwd_weight_workspace_bytes(N, C, H, W, K, dtype);
  if (workspace_bytes < need || (need > 0 && !workspace))
    return fail(O1D_ERR_WORKSPACE, "%s: workspace of %zu bytes given, %zu needed", fn, workspace_bytes, need);
  const size_t dwbytes = (size_t)C * K * elem_size(dtype), tbytes = elems * elem_size(dtype);
  if (overlaps(dw, dwbytes, x, tbytes) || overlaps(dw, dwbytes, dy, tbytes) ||
      (need > 0 && (overlaps(workspace, need, x, tbytes) || overlaps(workspace, need, dy, tbytes) ||
                    overlaps(workspace, need, dw, dwbytes))))
    return fail(O1D_ERR_INVALID, "%s: dw or workspace overlaps an input", fn);
  return wgrad_dispatch(fn, x, dy, theta_deg, dw, N, C, H, W, K, dtype, workspace, s);
}

o1d_status_t o1d_bwd(const void* x, const void* dy, const void* w, const float* theta_deg, void* dx, void* dw, int N,
                     int C, int H, int W, int K, o1d_dtype_t dtype, void* workspace, size_t workspace_bytes,
                     void* stream) {
  const char* fn = "o1d_bwd";
  o1d_status_t st = check_sizes(fn, N, C, H, W, K, dtype);
  if (st != O1D_OK) return st;
  if (C == 0) return ok();
  if (!dw) return fail(O1D_ERR_INVALID, "%s: NULL dw pointer", fn);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t elems = (size_t)N * C * H * W;
  (void)hipGetLastError();
  if (elems == 0) return hip_status(fn, o1d::launch_zero((o1d::Dtype)dtype, dw, (size_t)C * K, s));
  if (!x || !dy || !w || !theta_deg || !dx) return fail(O1D_ERR_INVALID, "%s: NULL tensor pointer", fn);
  const size_t need = o1d_bwd_weight_workspace_bytes(N, C, H, W, K, dtype);
  if (workspace_bytes < need || (need > 0 && !workspace))
    return fail(O1D_ERR_WORKSPACE, "%s: workspace of %zu bytes given, %zu needed", fn, workspace_bytes, need);
  const size_t wbytes = (size_t)C * K * elem_size(dtype), tbytes = elems * elem_size(dtype);
  if (overlaps(dx, tbytes, x, tbytes) || overlaps(dx, tbytes, dy, tbytes) || overlaps(dx, tbytes, w, wbytes))
    return fail(O1D_ERR_INVALID, "%s: dx overlaps an input", fn);
  if (overlaps(dw, wbytes, x, tbytes) || overlaps(dw, wbytes, dy, tbytes) || overlaps(dw, wbytes, w, wbytes) ||
      overlaps(dw, wbytes, dx, tbytes))
    return fail(O1D_ERR_INVALID, "%s: dw overlaps an input or dx", fn);
  if (need > 0 && (overlaps(workspace, need, x, tbytes) || overlaps(workspace, need, dy, tbytes) ||
                   overlaps(workspace, need, w, wbytes) || overlaps(workspace, need, dx, tbytes) ||
                   overlaps(workspace, need, dw, wbytes)))
    return fail(O1D_ERR_INVALID, "%s: workspace overlaps a tensor", fn);
  const bool va = vec_aligned(x, dtype) && vec_aligned(dy, dtype) && vec_aligned(dx, dtype);
  if (line_allowed()) {
    // the weight gradient's plan (hence its workspace) with mirrored offsets
    o1d::strip::Plan sp = o1d::strip::plan_strip(N, C, H, W, K, -1, 1, va);
    if (sp.ok)
      return hip_status(fn, o1d::launch_bwd_strip((o1d::Dtype)dtype, sp, x, dy, w, theta_deg, dx, dw,
                                                  static_cast<float*>(workspace), s));
  }
  st = gather_entry(fn, dy, w, theta_deg, dx, N, C, H, W, K, dtype, stream, -1);
  if (st != O1D_OK) return st;
  return wgrad_dispatch(fn, x, dy, theta_deg, dw, N, C, H, W, K, dtype, workspace, s);
}

const char* o1d_status_str(o1d_status_t status) {
  switch (status) {
    case O1D_OK: return "O1D_OK";
    case O1D_ERR_INVALID: return "O1D_ERR_INVALID: invalid argument";
    case O1D_ERR_UNSUPPORTED: return "O1D_ERR_UNSUPPORTED: size outside the supported range";
    case O1D_ERR_WORKSPACE: return "O1D_ERR_WORKSPACE: workspace too small";
    case O1D_ERR_HIP: return "O1D_ERR_HIP: HIP runtime error";
  }
  return "unknown o1d status";
}

const char* o1d_last_error(void) { return g_last_error; }

const char* o1d_version(void) { return "o1d 0.1.0 (gfx950)"; }

}  // extern "C"
