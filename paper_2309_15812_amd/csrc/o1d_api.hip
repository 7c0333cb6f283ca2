// C ABI of the oriented 1D depthwise convolution library (declared in
// include/o1d.h): argument validation, status codes, per-thread error text,
// the choice of kernel family and dispatch to the launchers.  No device
// memory is allocated here.
//
// Kernel families:
//  * strip kernels (o1d_strip*.h): NCHW, stride 1, offsets rounded down,
//    W a multiple of 4, vector-aligned tensors, planes whose zero-margined
//    tile fits the compiled tile strides; gathers for K <= 63, the weight
//    gradient and the fused backward for K <= 31;
//  * plane kernels (o1d_plane*.h): NCHW planes small enough that a whole
//    plane, for a group of images, fits in LDS (lanes over images; any
//    stride, both discretisations, the fused backward at stride 1 rounding
//    down);
//  * general kernels (o1d_gen*.h): everything else the ABI accepts;
//  * the depthwise separable block adds the pointwise convolution's matrix
//    products on the matrix cores (o1d_pw*.h).
#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>

#include "o1d.h"
#include "o1d_gen.h"
#include "o1d_launch.h"
#include "o1d_plane.h"
#include "o1d_pw.h"
#include "o1d_strip.h"

namespace {

thread_local char g_last_error[512] = "";
thread_local char g_name[256] = "";

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
const char* dt_name(o1d_dtype_t dt) { return dt == O1D_BF16 ? "bf16" : "f32"; }

bool overlaps(const void* a, size_t abytes, const void* b, size_t bbytes) {
  const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + bbytes && b0 < a0 + abytes;
}

// The options every entry point takes (the plain entry points: stride 1,
// NCHW, rounding down).
struct Opts {
  int stride = 1;
  o1d_layout_t layout = O1D_NCHW;
  o1d_sampling_t sampling = O1D_FLOOR;
  bool plain() const { return stride == 1 && layout == O1D_NCHW && sampling == O1D_FLOOR; }
};

// Checks shared by all entry points.
o1d_status_t check_sizes(const char* fn, int N, int C, int H, int W, int K, o1d_dtype_t dt, const Opts& o) {
  if (dt != O1D_F32 && dt != O1D_BF16) return fail(O1D_ERR_INVALID, "%s: unknown dtype %d", fn, (int)dt);
  if (N < 0 || C < 0 || H < 0 || W < 0)
    return fail(O1D_ERR_INVALID, "%s: negative size N=%d C=%d H=%d W=%d", fn, N, C, H, W);
  if (K < 1 || (K % 2) == 0)
    return fail(O1D_ERR_INVALID, "%s: K=%d must be odd and positive (pad = K/2 centres the kernel)", fn, K);
  if (o.stride < 1) return fail(O1D_ERR_INVALID, "%s: stride %d must be >= 1", fn, o.stride);
  if (o.layout != O1D_NCHW && o.layout != O1D_NHWC)
    return fail(O1D_ERR_INVALID, "%s: unknown layout %d", fn, (int)o.layout);
  if (o.sampling != O1D_FLOOR && o.sampling != O1D_BILINEAR)
    return fail(O1D_ERR_INVALID, "%s: unknown sampling %d", fn, (int)o.sampling);
  if (K > O1D_MAX_K) return fail(O1D_ERR_UNSUPPORTED, "%s: K=%d exceeds O1D_MAX_K=%d", fn, K, O1D_MAX_K);
  if (o.stride > 64) return fail(O1D_ERR_UNSUPPORTED, "%s: stride %d exceeds 64", fn, o.stride);
  if (C > 65535 || N > 65535)
    return fail(O1D_ERR_UNSUPPORTED, "%s: N=%d or C=%d exceeds the 65535 grid limit", fn, N, C);
  if ((long long)N * C * (long long)H * W >= (1ll << 31))
    return fail(O1D_ERR_UNSUPPORTED, "%s: %d x %d x %d x %d elements exceed 2^31", fn, N, C, H, W);
  return O1D_OK;
}

// Vector staging needs 16-byte (float32) or 8-byte (bfloat16) aligned tensors.
bool vec_aligned(const void* p, o1d_dtype_t dt) { return ((uintptr_t)p % (dt == O1D_BF16 ? 8u : 16u)) == 0; }

enum OpKind { kOpFwd = 0, kOpDgrad = 1, kOpWgrad = 2, kOpBwd = 3 };

// The kernels one op runs: the strip kernels where they apply, else the
// plane kernels, else the general kernels.  For the fused backward (kOpBwd)
// the route is a one-pass kernel of the same order; where none applies (the
// route is not ok) o1d_bwd runs the input gradient's route and then the
// weight gradient's.
enum class Family { None, Strip, Plane, Gen };

struct Route {
  bool ok = false;
  Family fam = Family::None;
  o1d::strip::Plan sp;
  o1d::plane::Plan pp;
  o1d::gen::Plan gp;
};

Route route(int op, int N, int C, int H, int W, int K, o1d_dtype_t dt, const Opts& o, bool aligned) {
  Route r;
  if (op == kOpBwd && !o.plain()) return r;
  if (o.plain()) {
    // the fused backward has the weight gradient's strip plan
    r.sp = o1d::strip::plan_strip(N, C, H, W, K, op == kOpDgrad || op == kOpBwd ? -1 : 1,
                                  op == kOpWgrad ? 1 : (op == kOpBwd ? 2 : 0), aligned);
    if (r.sp.ok) {
      r.ok = true;
      r.fam = Family::Strip;
      return r;
    }
  }
  const int sampling = o.sampling == O1D_BILINEAR ? 1 : 0;
  if (o.layout == O1D_NCHW) {
    r.pp = o1d::plane::plan_plane(op, N, C, H, W, K, o.stride, sampling, (int)elem_size(dt), aligned);
    if (r.pp.ok) {
      r.ok = true;
      r.fam = Family::Plane;
      return r;
    }
  }
  const int gop = op == kOpFwd ? o1d::gen::kFwd
                               : (op == kOpDgrad ? o1d::gen::kDgrad : (op == kOpWgrad ? o1d::gen::kWgrad : o1d::gen::kBwd));
  r.gp = o1d::gen::plan_gen(gop, o.layout == O1D_NHWC ? o1d::gen::kNHWC : o1d::gen::kNCHW, N, C, H, W, K, o.stride,
                            sampling, (int)elem_size(dt));
  if (r.gp.ok) {
    r.ok = true;
    r.fam = Family::Gen;
  }
  return r;
}

// Partial rows per channel of the weight gradient's route.
size_t route_parts(const Route& r) {
  switch (r.fam) {
    case Family::Strip: return (size_t)r.sp.blocks_n;
    case Family::Plane: return r.pp.parts;
    case Family::Gen: return r.gp.parts;
    default: return 0;
  }
}

// The weight gradient's workspace holds one partial row of K float32 per
// channel and workgroup.  Its size must not depend on pointer alignment, so
// the larger partial count of the aligned and unaligned routes is reported
// (the fused backward's strip plan has the weight gradient's partial count).
size_t wgrad_workspace(int N, int C, int H, int W, int K, o1d_dtype_t dt, const Opts& o) {
  size_t parts = 0;
  for (int a = 0; a < 2; ++a)
    for (int op : {kOpWgrad, kOpBwd}) {
      const Route r = route(op, N, C, H, W, K, dt, o, a != 0);
      if (r.ok && route_parts(r) > parts) parts = route_parts(r);
    }
  return parts * (size_t)C * (size_t)K * sizeof(float);
}

o1d_status_t hip_status(const char* fn, hipError_t e) {
  if (e != hipSuccess) return fail(O1D_ERR_HIP, "%s: kernel launch failed: %s", fn, hipGetErrorString(e));
  return ok();
}

o1d_status_t unsupported(const char* fn, int N, int C, int H, int W, int K) {
  return fail(O1D_ERR_UNSUPPORTED, "%s: no kernel covers N=%d C=%d H=%d W=%d K=%d (LDS tile too large)", fn, N, C, H,
              W, K);
}

// Tensor sizes of the op's tensors in elements: input plane and output plane.
size_t in_elems(int N, int C, int H, int W) { return (size_t)N * C * H * W; }
size_t out_elems(int N, int C, int H, int W, int s) {
  return (size_t)N * C * (size_t)o1d::gen::out_size(H, s) * (size_t)o1d::gen::out_size(W, s);
}

// Forward (sign +1: x -> y) or input gradient (sign -1: dy -> dx) after the
// size checks.  H and W are always the input plane's.
o1d_status_t gather_entry(const char* fn, const void* in, const void* w, const float* theta, void* out, int N, int C,
                          int H, int W, int K, o1d_dtype_t dt, const Opts& o, void* stream, int sign) {
  o1d_status_t st = check_sizes(fn, N, C, H, W, K, dt, o);
  if (st != O1D_OK) return st;
  if (in_elems(N, C, H, W) == 0) return ok();
  if (!in || !w || !theta || !out) return fail(O1D_ERR_INVALID, "%s: NULL tensor pointer", fn);
  const size_t xb = in_elems(N, C, H, W) * elem_size(dt), yb = out_elems(N, C, H, W, o.stride) * elem_size(dt);
  const size_t inb = sign > 0 ? xb : yb, outb = sign > 0 ? yb : xb;
  if (overlaps(in, inb, out, outb)) return fail(O1D_ERR_INVALID, "%s: output overlaps input", fn);
  (void)hipGetLastError();
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool va = vec_aligned(in, dt) && vec_aligned(out, dt);
  const Route r = route(sign > 0 ? kOpFwd : kOpDgrad, N, C, H, W, K, dt, o, va);
  if (!r.ok) return unsupported(fn, N, C, H, W, K);
  if (r.fam == Family::Strip)
    return hip_status(fn, o1d::launch_gather_strip((o1d::Dtype)dt, r.sp, in, w, theta, out, s));
  if (r.fam == Family::Plane)
    return hip_status(fn, o1d::launch_plane_gather((o1d::Dtype)dt, r.pp, in, w, theta, out, s));
  return hip_status(fn, o1d::launch_gen_gather((o1d::Dtype)dt, r.gp, (int)o.layout, in, w, theta, out, s));
}

// Weight gradient after validation.
o1d_status_t wgrad_dispatch(const char* fn, const void* x, const void* dy, const float* theta, void* dw, int N, int C,
                            int H, int W, int K, o1d_dtype_t dt, const Opts& o, void* workspace, hipStream_t s) {
  const bool va = vec_aligned(x, dt) && vec_aligned(dy, dt);
  const Route r = route(kOpWgrad, N, C, H, W, K, dt, o, va);
  if (!r.ok) return unsupported(fn, N, C, H, W, K);
  float* part = static_cast<float*>(workspace);
  if (r.fam == Family::Strip)
    return hip_status(fn, o1d::launch_wgrad_strip((o1d::Dtype)dt, r.sp, x, dy, theta, dw, part, s));
  if (r.fam == Family::Plane)
    return hip_status(fn, o1d::launch_plane_wgrad((o1d::Dtype)dt, r.pp, x, dy, theta, dw, part, s));
  return hip_status(fn, o1d::launch_gen_wgrad((o1d::Dtype)dt, r.gp, (int)o.layout, x, dy, theta, dw, part, s));
}

o1d_status_t bwd_weight_entry(const char* fn, const void* x, const void* dy, const float* theta_deg, void* dw, int N,
                              int C, int H, int W, int K, o1d_dtype_t dtype, const Opts& o, void* workspace,
                              size_t workspace_bytes, void* stream) {
  o1d_status_t st = check_sizes(fn, N, C, H, W, K, dtype, o);
  if (st != O1D_OK) return st;
  if (C == 0) return ok();
  if (!dw) return fail(O1D_ERR_INVALID, "%s: NULL dw pointer", fn);
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  if (in_elems(N, C, H, W) == 0) return hip_status(fn, o1d::launch_zero((o1d::Dtype)dtype, dw, (size_t)C * K, s));
  if (!x || !dy || !theta_deg) return fail(O1D_ERR_INVALID, "%s: NULL tensor pointer", fn);
  const size_t need = wgrad_workspace(N, C, H, W, K, dtype, o);
  if (need == 0) return unsupported(fn, N, C, H, W, K);
  if (workspace_bytes < need || !workspace)
    return fail(O1D_ERR_WORKSPACE, "%s: workspace of %zu bytes given, %zu needed", fn, workspace_bytes, need);
  const size_t dwb = (size_t)C * K * elem_size(dtype), xb = in_elems(N, C, H, W) * elem_size(dtype);
  const size_t yb = out_elems(N, C, H, W, o.stride) * elem_size(dtype);
  if (overlaps(dw, dwb, x, xb) || overlaps(dw, dwb, dy, yb) || overlaps(workspace, need, x, xb) ||
      overlaps(workspace, need, dy, yb) || overlaps(workspace, need, dw, dwb))
    return fail(O1D_ERR_INVALID, "%s: dw or workspace overlaps an input", fn);
  return wgrad_dispatch(fn, x, dy, theta_deg, dw, N, C, H, W, K, dtype, o, workspace, s);
}

void name_of(char* buf, size_t n, int op, const Route& r, o1d_dtype_t dt, const Opts& o) {
  static const char* fam[] = {"gather", "gather", "wgrad", "bwd"};
  if (r.fam == Family::Strip)
    snprintf(buf, n, "strip_%s/%s/S%d/KB%d", fam[op], dt_name(dt), r.sp.S, r.sp.KB);
  else if (r.fam == Family::Plane)
    snprintf(buf, n, "plane_%s/%s/RP%d%s", fam[op], dt_name(dt), r.pp.p.RP,
             op >= kOpWgrad ? (r.pp.p.KB == 32 ? "/KB32" : (r.pp.p.KB == 64 ? "/KB64" : "/KB128")) : "");
  else
    snprintf(buf, n, "gen_%s/%s/%s/RP%d%s", fam[op], dt_name(dt), o.layout == O1D_NHWC ? "nhwc" : "nchw", r.gp.p.RP,
             op >= kOpWgrad ? (r.gp.p.KB == 32 ? "/KB32" : (r.gp.p.KB == 64 ? "/KB64" : "/KB128")) : "");
}

o1d_status_t bwd_entry(const char* fn, const void* x, const void* dy, const void* w, const float* theta_deg,
                       void* dx, void* dw, int N, int C, int H, int W, int K, o1d_dtype_t dtype, void* workspace,
                       size_t workspace_bytes, void* stream) {
  const Opts o;
  o1d_status_t st = check_sizes(fn, N, C, H, W, K, dtype, o);
  if (st != O1D_OK) return st;
  if (C == 0) return ok();
  if (!dw) return fail(O1D_ERR_INVALID, "%s: NULL dw pointer", fn);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t elems = in_elems(N, C, H, W);
  (void)hipGetLastError();
  if (elems == 0) return hip_status(fn, o1d::launch_zero((o1d::Dtype)dtype, dw, (size_t)C * K, s));
  if (!x || !dy || !w || !theta_deg || !dx) return fail(O1D_ERR_INVALID, "%s: NULL tensor pointer", fn);
  const size_t need = wgrad_workspace(N, C, H, W, K, dtype, o);
  if (need == 0) return unsupported(fn, N, C, H, W, K);
  if (workspace_bytes < need || !workspace)
    return fail(O1D_ERR_WORKSPACE, "%s: workspace of %zu bytes given, %zu needed", fn, workspace_bytes, need);
  const size_t wbytes = (size_t)C * K * elem_size(dtype), tbytes = elems * elem_size(dtype);
  if (overlaps(dx, tbytes, x, tbytes) || overlaps(dx, tbytes, dy, tbytes) || overlaps(dx, tbytes, w, wbytes))
    return fail(O1D_ERR_INVALID, "%s: dx overlaps an input", fn);
  if (overlaps(dw, wbytes, x, tbytes) || overlaps(dw, wbytes, dy, tbytes) || overlaps(dw, wbytes, w, wbytes) ||
      overlaps(dw, wbytes, dx, tbytes))
    return fail(O1D_ERR_INVALID, "%s: dw overlaps an input or dx", fn);
  if (overlaps(workspace, need, x, tbytes) || overlaps(workspace, need, dy, tbytes) ||
      overlaps(workspace, need, w, wbytes) || overlaps(workspace, need, dx, tbytes) ||
      overlaps(workspace, need, dw, wbytes))
    return fail(O1D_ERR_INVALID, "%s: workspace overlaps a tensor", fn);
  const bool va = vec_aligned(x, dtype) && vec_aligned(dy, dtype) && vec_aligned(dx, dtype);
  const Route r = route(kOpBwd, N, C, H, W, K, dtype, o, va);
  float* part = static_cast<float*>(workspace);
  if (r.fam == Family::Strip)
    return hip_status(fn, o1d::launch_bwd_strip((o1d::Dtype)dtype, r.sp, x, dy, w, theta_deg, dx, dw, part, s));
  if (r.fam == Family::Plane)
    return hip_status(fn, o1d::launch_plane_bwd((o1d::Dtype)dtype, r.pp, x, dy, w, theta_deg, dx, dw, part, s));
  if (r.fam == Family::Gen)
    return hip_status(fn, o1d::launch_gen_bwd((o1d::Dtype)dtype, r.gp, x, dy, w, theta_deg, dx, dw, part, s));
  st = gather_entry(fn, dy, w, theta_deg, dx, N, C, H, W, K, dtype, o, stream, -1);
  if (st != O1D_OK) return st;
  return wgrad_dispatch(fn, x, dy, theta_deg, dw, N, C, H, W, K, dtype, o, workspace, s);
}


// ---- depthwise separable block: the pointwise convolution's products

enum PwKind { kPwFwd = 0, kPwDgrad = 1, kPwWgrad = 2 };

// The strided batched product of one pointwise step (see o1d_pw.h); the
// weight gradient sums the images in groups sized so that about 1024
// workgroups run.
o1d::pw::Params pw_params(int kind, int N, int C, int Cout, int H, int W) {
  o1d::pw::Params p{};
  const int HW = H * W;
  p.nbatch = N;
  if (kind == kPwFwd) {  // Y_n = Wp Z_n
    p.M = Cout; p.N = HW; p.K = C;
    p.sA = 0; p.am = C; p.ak = 1; p.a_kc = 1;
    p.sB = (long long)C * HW; p.bk = HW; p.bn = 1; p.b_nc = 1;
    p.sC = (long long)Cout * HW; p.cm = HW; p.cn = 1;
  } else if (kind == kPwDgrad) {  // dZ_n = Wp^T dY_n
    p.M = C; p.N = HW; p.K = Cout;
    p.sA = 0; p.am = 1; p.ak = C; p.a_kc = 0;
    p.sB = (long long)Cout * HW; p.bk = HW; p.bn = 1; p.b_nc = 1;
    p.sC = (long long)C * HW; p.cm = HW; p.cn = 1;
  } else {  // dWp = sum_n dY_n Z_n^T
    p.M = Cout; p.N = C; p.K = HW;
    p.sA = (long long)Cout * HW; p.am = HW; p.ak = 1; p.a_kc = 1;
    p.sB = (long long)C * HW; p.bk = 1; p.bn = HW; p.b_nc = 0;
    p.sC = 0; p.cm = C; p.cn = 1;
    p.sum = 1;
  }
  p.tm = o1d::pw::cdiv(p.M, o1d::pw::kBM);
  p.tn = o1d::pw::cdiv(p.N, o1d::pw::kBN);
  if (p.sum) {
    const int tiles = p.tm * p.tn;
    int nsplit = std::min(N, std::max(1, o1d::pw::cdiv(1024, tiles)));
    p.per_split = o1d::pw::cdiv(N, nsplit);
    p.nsplit = o1d::pw::cdiv(N, p.per_split);
  }
  return p;
}

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

// The backward's workspace: dz, the pointwise weight gradient's partials,
// the depthwise backward's workspace.
struct DscWorkspace {
  size_t dz = 0, part = 0, dw = 0, total = 0;
};

DscWorkspace dsc_workspace(int N, int C, int Cout, int H, int W, int K, o1d_dtype_t dt) {
  DscWorkspace ws;
  const o1d::pw::Params pg = pw_params(kPwWgrad, N, C, Cout, H, W);
  ws.dz = align256(in_elems(N, C, H, W) * elem_size(dt));
  ws.part = align256((size_t)pg.nsplit * Cout * C * sizeof(float));
  ws.dw = wgrad_workspace(N, C, H, W, K, dt, Opts());
  ws.total = ws.dz + ws.part + ws.dw;
  return ws;
}

o1d_status_t check_cout(const char* fn, int Cout) {
  if (Cout < 1 || Cout > 65535) return fail(O1D_ERR_INVALID, "%s: Cout=%d must be 1 .. 65535", fn, Cout);
  return O1D_OK;
}

// ---- fixed scratch of the no-allocation entry point (o1d_bwd_noalloc)
//
// The weight gradient's partial rows live in a file-scope device array
// instead of a caller workspace.  Each GPU holds its own copy; its address
// is looked up once per device (with that device current) and kept, and
// host code only ever uses that address, never the array's name.  Every
// call on a GPU shares the array, so calls that overlap on one GPU race.
// Nothing needs clearing: every workgroup overwrites its whole partial row
// before the reduction reads it.
constexpr size_t kScratchBytes = (size_t)8 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

o1d_status_t scratch_ptr(const char* fn, void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(O1D_ERR_HIP, "%s: hipGetDevice failed: %s", fn, hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(O1D_ERR_UNSUPPORTED, "%s: device %d out of range", fn, dev);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(O1D_ERR_HIP, "%s: hipGetSymbolAddress of the scratch failed: %s", fn, hipGetErrorString(e));
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return O1D_OK;
}

}  // namespace

extern "C" {

size_t o1d_bwd_weight_workspace_bytes(int N, int C, int H, int W, int K, o1d_dtype_t dtype) {
  const Opts o;
  if (check_sizes("o1d_bwd_weight_workspace_bytes", N, C, H, W, K, dtype, o) != O1D_OK) return 0;
  if (in_elems(N, C, H, W) == 0) return 0;
  return wgrad_workspace(N, C, H, W, K, dtype, o);
}

size_t o1d_bwd_weight_ex_workspace_bytes(int N, int C, int H, int W, int K, int stride, o1d_layout_t layout,
                                         o1d_sampling_t sampling, o1d_dtype_t dtype) {
  Opts o;
  o.stride = stride;
  o.layout = layout;
  o.sampling = sampling;
  if (check_sizes("o1d_bwd_weight_ex_workspace_bytes", N, C, H, W, K, dtype, o) != O1D_OK) return 0;
  if (in_elems(N, C, H, W) == 0) return 0;
  return wgrad_workspace(N, C, H, W, K, dtype, o);
}

o1d_status_t o1d_fwd(const void* x, const void* w, const float* theta_deg, void* y, int N, int C, int H, int W, int K,
                     o1d_dtype_t dtype, void* stream) {
  return gather_entry("o1d_fwd", x, w, theta_deg, y, N, C, H, W, K, dtype, Opts(), stream, +1);
}

o1d_status_t o1d_bwd_input(const void* dy, const void* w, const float* theta_deg, void* dx, int N, int C, int H,
                           int W, int K, o1d_dtype_t dtype, void* stream) {
  return gather_entry("o1d_bwd_input", dy, w, theta_deg, dx, N, C, H, W, K, dtype, Opts(), stream, -1);
}

o1d_status_t o1d_bwd_weight(const void* x, const void* dy, const float* theta_deg, void* dw, int N, int C, int H,
                            int W, int K, o1d_dtype_t dtype, void* workspace, size_t workspace_bytes, void* stream) {
  return bwd_weight_entry("o1d_bwd_weight", x, dy, theta_deg, dw, N, C, H, W, K, dtype, Opts(), workspace,
                          workspace_bytes, stream);
}

o1d_status_t o1d_fwd_ex(const void* x, const void* w, const float* theta_deg, void* y, int N, int C, int H, int W,
                        int K, int stride, o1d_layout_t layout, o1d_sampling_t sampling, o1d_dtype_t dtype,
                        void* stream) {
  Opts o;
  o.stride = stride;
  o.layout = layout;
  o.sampling = sampling;
  return gather_entry("o1d_fwd_ex", x, w, theta_deg, y, N, C, H, W, K, dtype, o, stream, +1);
}

o1d_status_t o1d_bwd_input_ex(const void* dy, const void* w, const float* theta_deg, void* dx, int N, int C, int H,
                              int W, int K, int stride, o1d_layout_t layout, o1d_sampling_t sampling,
                              o1d_dtype_t dtype, void* stream) {
  Opts o;
  o.stride = stride;
  o.layout = layout;
  o.sampling = sampling;
  return gather_entry("o1d_bwd_input_ex", dy, w, theta_deg, dx, N, C, H, W, K, dtype, o, stream, -1);
}

o1d_status_t o1d_bwd_weight_ex(const void* x, const void* dy, const float* theta_deg, void* dw, int N, int C, int H,
                               int W, int K, int stride, o1d_layout_t layout, o1d_sampling_t sampling,
                               o1d_dtype_t dtype, void* workspace, size_t workspace_bytes, void* stream) {
  Opts o;
  o.stride = stride;
  o.layout = layout;
  o.sampling = sampling;
  return bwd_weight_entry("o1d_bwd_weight_ex", x, dy, theta_deg, dw, N, C, H, W, K, dtype, o, workspace,
                          workspace_bytes, stream);
}

o1d_status_t o1d_bwd(const void* x, const void* dy, const void* w, const float* theta_deg, void* dx, void* dw, int N,
                     int C, int H, int W, int K, o1d_dtype_t dtype, void* workspace, size_t workspace_bytes,
                     void* stream) {
  return bwd_entry("o1d_bwd", x, dy, w, theta_deg, dx, dw, N, C, H, W, K, dtype, workspace, workspace_bytes, stream);
}

o1d_status_t o1d_bwd_noalloc(const void* x, const void* dy, const void* w, const float* theta_deg, void* dx,
                             void* dw, int N, int C, int H, int W, int K, o1d_dtype_t dtype, void* stream) {
  const char* fn = "o1d_bwd_noalloc";
  const Opts o;
  o1d_status_t st = check_sizes(fn, N, C, H, W, K, dtype, o);
  if (st != O1D_OK) return st;
  if (C == 0 || in_elems(N, C, H, W) == 0)
    return bwd_entry(fn, x, dy, w, theta_deg, dx, dw, N, C, H, W, K, dtype, nullptr, 0, stream);
  const size_t need = wgrad_workspace(N, C, H, W, K, dtype, o);
  if (need > kScratchBytes)
    return fail(O1D_ERR_UNSUPPORTED, "%s: these sizes need %zu bytes of scratch; the fixed scratch holds %zu", fn,
                need, kScratchBytes);
  void* ptr = nullptr;
  st = scratch_ptr(fn, &ptr);
  if (st != O1D_OK) return st;
  return bwd_entry(fn, x, dy, w, theta_deg, dx, dw, N, C, H, W, K, dtype, ptr, kScratchBytes, stream);
}

o1d_status_t o1d_dsc_fwd(const void* x, const void* w_dw, const float* theta_deg, const void* w_pw, void* z,
                         void* y, int N, int C, int Cout, int H, int W, int K, o1d_dtype_t dtype, void* stream) {
  const char* fn = "o1d_dsc_fwd";
  const Opts o;
  o1d_status_t st = check_sizes(fn, N, C, H, W, K, dtype, o);
  if (st != O1D_OK) return st;
  if ((st = check_cout(fn, Cout)) != O1D_OK) return st;
  const size_t pix = (size_t)N * H * W;
  if (pix == 0) return ok();
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t yb = pix * Cout * elem_size(dtype), zb = in_elems(N, C, H, W) * elem_size(dtype);
  if (!y) return fail(O1D_ERR_INVALID, "%s: NULL y pointer", fn);
  (void)hipGetLastError();
  if (C == 0) return hip_status(fn, o1d::launch_zero((o1d::Dtype)dtype, y, pix * Cout, s));
  if (!x || !w_dw || !theta_deg || !w_pw || !z) return fail(O1D_ERR_INVALID, "%s: NULL tensor pointer", fn);
  const size_t xb = zb, wpb = (size_t)Cout * C * elem_size(dtype);
  if (overlaps(y, yb, x, xb) || overlaps(y, yb, z, zb) || overlaps(y, yb, w_pw, wpb) || overlaps(z, zb, w_pw, wpb))
    return fail(O1D_ERR_INVALID, "%s: y or z overlaps another tensor", fn);
  st = gather_entry(fn, x, w_dw, theta_deg, z, N, C, H, W, K, dtype, o, stream, +1);
  if (st != O1D_OK) return st;
  return hip_status(fn, o1d::launch_pw_gemm((o1d::Dtype)dtype, pw_params(kPwFwd, N, C, Cout, H, W), w_pw, z, y, s));
}

size_t o1d_dsc_bwd_workspace_bytes(int N, int C, int Cout, int H, int W, int K, o1d_dtype_t dtype) {
  const Opts o;
  if (check_sizes("o1d_dsc_bwd_workspace_bytes", N, C, H, W, K, dtype, o) != O1D_OK) return 0;
  if (check_cout("o1d_dsc_bwd_workspace_bytes", Cout) != O1D_OK) return 0;
  if (in_elems(N, C, H, W) == 0) return 0;
  return dsc_workspace(N, C, Cout, H, W, K, dtype).total;
}

o1d_status_t o1d_dsc_bwd(const void* x, const void* z, const void* dy, const void* w_dw, const float* theta_deg,
                         const void* w_pw, void* dx, void* dw_dw, void* dw_pw, int N, int C, int Cout, int H,
                         int W, int K, o1d_dtype_t dtype, void* workspace, size_t workspace_bytes, void* stream) {
  const char* fn = "o1d_dsc_bwd";
  const Opts o;
  o1d_status_t st = check_sizes(fn, N, C, H, W, K, dtype, o);
  if (st != O1D_OK) return st;
  if ((st = check_cout(fn, Cout)) != O1D_OK) return st;
  if (C == 0) return ok();
  if (!dw_dw || !dw_pw) return fail(O1D_ERR_INVALID, "%s: NULL weight-gradient pointer", fn);
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  const size_t elems = in_elems(N, C, H, W);
  if (elems == 0) {
    st = hip_status(fn, o1d::launch_zero((o1d::Dtype)dtype, dw_dw, (size_t)C * K, s));
    if (st != O1D_OK) return st;
    return hip_status(fn, o1d::launch_zero((o1d::Dtype)dtype, dw_pw, (size_t)Cout * C, s));
  }
  if (!x || !z || !dy || !w_dw || !theta_deg || !w_pw || !dx) return fail(O1D_ERR_INVALID, "%s: NULL tensor pointer", fn);
  const DscWorkspace ws = dsc_workspace(N, C, Cout, H, W, K, dtype);
  if (workspace_bytes < ws.total || !workspace)
    return fail(O1D_ERR_WORKSPACE, "%s: workspace of %zu bytes given, %zu needed", fn, workspace_bytes, ws.total);
  const size_t es = elem_size(dtype), tb = elems * es, yb = (size_t)N * Cout * H * W * es;
  const size_t wpb = (size_t)Cout * C * es, wdb = (size_t)C * K * es;
  const void* ins[] = {x, z, dy, w_dw, w_pw};
  const size_t inb[] = {tb, tb, yb, wdb, wpb};
  void* outs[] = {dx, dw_dw, dw_pw, workspace};
  const size_t outb[] = {tb, wdb, wpb, ws.total};
  for (int i = 0; i < 4; ++i) {
    for (int j = 0; j < 5; ++j)
      if (overlaps(outs[i], outb[i], ins[j], inb[j])) return fail(O1D_ERR_INVALID, "%s: an output overlaps an input", fn);
    for (int j = i + 1; j < 4; ++j)
      if (overlaps(outs[i], outb[i], outs[j], outb[j])) return fail(O1D_ERR_INVALID, "%s: outputs overlap", fn);
  }
  unsigned char* wsb = static_cast<unsigned char*>(workspace);
  void* dz = wsb;
  float* part = reinterpret_cast<float*>(wsb + ws.dz);
  void* dws = wsb + ws.dz + ws.part;
  st = hip_status(fn, o1d::launch_pw_gemm((o1d::Dtype)dtype, pw_params(kPwDgrad, N, C, Cout, H, W), w_pw, dy, dz, s));
  if (st != O1D_OK) return st;
  const o1d::pw::Params pg = pw_params(kPwWgrad, N, C, Cout, H, W);
  st = hip_status(fn, o1d::launch_pw_gemm((o1d::Dtype)dtype, pg, dy, z, part, s));
  if (st != O1D_OK) return st;
  st = hip_status(fn, o1d::launch_partial_sum((o1d::Dtype)dtype, part, dw_pw, Cout * C, pg.nsplit, s));
  if (st != O1D_OK) return st;
  return bwd_entry(fn, x, dz, w_dw, theta_deg, dx, dw_dw, N, C, H, W, K, dtype, dws, ws.dw, stream);
}

const char* o1d_kernel_name(int op, int N, int C, int H, int W, int K, int stride, o1d_layout_t layout,
                            o1d_sampling_t sampling, o1d_dtype_t dtype, int aligned) {
  Opts o;
  o.stride = stride;
  o.layout = layout;
  o.sampling = sampling;
  g_name[0] = '\0';
  if (op < kOpFwd || op > kOpBwd || (op == kOpBwd && !o.plain())) return g_name;
  if (check_sizes("o1d_kernel_name", N, C, H, W, K, dtype, o) != O1D_OK || in_elems(N, C, H, W) == 0) return g_name;
  const Route r = route(op, N, C, H, W, K, dtype, o, aligned != 0);
  if (r.ok) {
    name_of(g_name, sizeof(g_name), op, r, dtype, o);
  } else if (op == kOpBwd) {
    char a[120], b[120];
    const Route rd = route(kOpDgrad, N, C, H, W, K, dtype, o, aligned != 0);
    const Route rw = route(kOpWgrad, N, C, H, W, K, dtype, o, aligned != 0);
    if (rd.ok && rw.ok) {
      name_of(a, sizeof(a), kOpDgrad, rd, dtype, o);
      name_of(b, sizeof(b), kOpWgrad, rw, dtype, o);
      snprintf(g_name, sizeof(g_name), "%s+%s", a, b);
    }
  }
  return g_name;
}

const char* o1d_kernel_variant(int i) {
  // every kernel instantiation compiled into the library, in the names
  // o1d_kernel_name uses
  struct Table {
    char names[192][48];
    int count = 0;
    Table() {
      for (const char* d : {"f32", "bf16"}) {
        for (int S : o1d::strip::kStrides) {
          snprintf(names[count++], 48, "strip_gather/%s/S%d/KB32", d, S);
          snprintf(names[count++], 48, "strip_gather/%s/S%d/KB64", d, S);
          snprintf(names[count++], 48, "strip_wgrad/%s/S%d/KB32", d, S);
          snprintf(names[count++], 48, "strip_bwd/%s/S%d/KB32", d, S);
        }
        for (const char* l : {"nchw", "nhwc"})
          for (int rp : {4, 8}) {
            snprintf(names[count++], 48, "gen_gather/%s/%s/RP%d", d, l, rp);
            for (int kb : {32, 64, 128}) {
              if (rp == 8 && kb != 32) continue;  // eight outputs per lane only with 32 sums
              snprintf(names[count++], 48, "gen_wgrad/%s/%s/RP%d/KB%d", d, l, rp, kb);
              if (l[1] == 'c') snprintf(names[count++], 48, "gen_bwd/%s/%s/RP%d/KB%d", d, l, rp, kb);
            }
          }
        for (int rp : {2, 4}) {
          snprintf(names[count++], 48, "plane_gather/%s/RP%d", d, rp);
          for (int kb : {32, 64, 128}) {
            snprintf(names[count++], 48, "plane_wgrad/%s/RP%d/KB%d", d, rp, kb);
            if (rp == 2 || kb != 128) snprintf(names[count++], 48, "plane_bwd/%s/RP%d/KB%d", d, rp, kb);
          }
        }
      }
    }
  };
  static const Table t;  // initialised once, thread-safe
  return i >= 0 && i < t.count ? t.names[i] : nullptr;
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

const char* o1d_version(void) { return "o1d 0.2.0 (gfx950)"; }

}  // extern "C"
