/*
 * o1d.h - C ABI of the MI355X (gfx950) library for depthwise convolution
 * with oriented 1D kernels.
 *
 * The operation is Definition 1, Eq. (1)-(2) of Kirchmeyer & Deng,
 * "Convolutional Networks with Oriented 1D Kernels" (ICCV 2023), with the
 * appendix "1D formulation" coordinate equation and the appendix "Padding"
 * rule (odd K, pad = K/2 inside the floor), stride 1 and zero padding:
 *
 *   y[n,c,p,q] = sum_{k=0}^{K-1} x[n,c, p + dh_c(k), q + dw_c(k)] * w[c,k]
 *   dh_c(k) = floor(-(k - K/2) * sin(theta_c)),
 *   dw_c(k) = floor( (k - K/2) * cos(theta_c)),
 *
 * where an x index outside [0,H) x [0,W) reads zero.  theta_c is given in
 * degrees; a product (k - K/2) * sin or cos that lies within 1e-9 of an
 * integer is taken to be that integer before the floor (so 0, 90, 30 ...
 * degrees give the exact-arithmetic offsets).  Taps that land on the same
 * pixel are summed.
 *
 * Layouts (all tensors dense, row-major, no strides):
 *   x, y, dy, dx : [N][C][H][W] in the element type `dtype`
 *   w, dw        : [C][K]       in the element type `dtype`
 *   theta_deg    : [C] float32 degrees, any finite value
 * Output size equals input size (P = H, Q = W).
 *
 * Memory and ownership: every tensor pointer is a DEVICE pointer owned by the
 * caller.  The library never allocates, frees or retains device memory on
 * these calls and keeps no per-call state, so calls are re-entrant.  All work
 * is enqueued asynchronously on `stream` (a hipStream_t; NULL selects the
 * null stream); the call returns after the enqueue.  Output buffers must not
 * alias input buffers.
 *
 * Precision: O1D_F32 computes and stores float32.  O1D_BF16 reads bfloat16,
 * accumulates in float32 and rounds the stored results to bfloat16 with
 * round-to-nearest-even.
 *
 * Errors: every argument check runs before any device work is enqueued; a
 * non-OK status means nothing was enqueued, except O1D_ERR_HIP, which reports
 * a failed kernel launch.  o1d_last_error() returns a human-readable detail
 * for the calling thread's most recent non-OK status.  Device faults, if
 * any, surface at the caller's next synchronisation.
 *
 * Empty tensors: a zero N, C, H or W is valid.  Nothing is launched, except
 * that o1d_bwd_weight and o1d_bwd with C > 0 write zeros to dw (an empty sum).
 */
#ifndef O1D_H_
#define O1D_H_

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  O1D_F32 = 0,  /* float32 storage and arithmetic */
  O1D_BF16 = 1  /* bfloat16 storage, float32 accumulation, RNE stores */
} o1d_dtype_t;

typedef enum {
  O1D_NCHW = 0, /* x[n][c][h][w] */
  O1D_NHWC = 1  /* x[n][h][w][c], Definition 1's own layout */
} o1d_layout_t;

typedef enum {
  O1D_FLOOR = 0,   /* Eq. (2): offsets rounded down */
  O1D_BILINEAR = 1 /* bilinear interpolation at the unrounded offsets (section "Discretization and
                      Interpolation"): tap k reads the four pixels around (str p + rh_k, str q + rw_k),
                      (rh_k, rw_k) = (-(k - K/2) sin theta, (k - K/2) cos theta), weighted by
                      (1-fh)(1-fw), (1-fh)fw, fh(1-fw), fh fw with fh, fw the fractional parts
                      (a part within 1e-9 of 0 or 1 is taken as 0 with the integer moved accordingly) */
} o1d_sampling_t;

typedef enum {
  O1D_OK = 0,
  O1D_ERR_INVALID = 1,     /* NULL pointer for a non-empty tensor, negative size, even or non-positive K,
                              unknown dtype, aliasing output */
  O1D_ERR_UNSUPPORTED = 2, /* K above O1D_MAX_K, a stride above 64, a size beyond the kernels' 32-bit index
                              range (2^31 elements, 65535 images or channels), or a zero-margined band of the
                              plane too large for LDS */
  O1D_ERR_WORKSPACE = 3,   /* workspace smaller than o1d_bwd_weight_workspace_bytes() */
  O1D_ERR_HIP = 4          /* the HIP runtime rejected a kernel launch */
} o1d_status_t;

#define O1D_MAX_K 127

/* Forward pass, Definition 1 / Eq. (1): y = conv(x; w, theta). */
o1d_status_t o1d_fwd(const void* x, const void* w, const float* theta_deg, void* y,
                     int N, int C, int H, int W, int K, o1d_dtype_t dtype, void* stream);

/* Gradient of Eq. (1) with respect to x (its adjoint in x):
 *   dx[n,c,h,w] = sum_k w[c,k] * dy[n,c, h - dh_c(k), w - dw_c(k)]   (zero outside the plane).
 * dx is overwritten, not accumulated. */
o1d_status_t o1d_bwd_input(const void* dy, const void* w, const float* theta_deg, void* dx,
                           int N, int C, int H, int W, int K, o1d_dtype_t dtype, void* stream);

/* Gradient of Eq. (1) with respect to w (its adjoint in w):
 *   dw[c,k] = sum_{n,p,q} dy[n,c,p,q] * x[n,c, p + dh_c(k), q + dw_c(k)]   (zero outside the plane).
 * dw is overwritten, not accumulated.  `workspace` is caller-owned device
 * memory of at least o1d_bwd_weight_workspace_bytes(...) bytes (may be NULL
 * when that size is 0); its contents on entry are ignored and are clobbered.
 * Partial sums are combined in a fixed order, so dw (like the outputs of
 * o1d_fwd and o1d_bwd_input) is bitwise reproducible for the same inputs. */
o1d_status_t o1d_bwd_weight(const void* x, const void* dy, const float* theta_deg, void* dw,
                            int N, int C, int H, int W, int K, o1d_dtype_t dtype,
                            void* workspace, size_t workspace_bytes, void* stream);

/* Both gradients of Eq. (1) in one call: dx as o1d_bwd_input computes it
 * (from dy and w) and dw as o1d_bwd_weight computes it (from x and dy).
 * One kernel reads x and dy once and produces both (then a small kernel adds
 * the weight gradient's partial rows); only where no one-pass kernel's LDS
 * tile fits (very large K with very wide planes) do the kernels of the two
 * separate entry points run in turn.  The results
 * equal those of the separate calls up to the order of floating-point
 * additions and are bitwise reproducible for the same inputs.  dx and dw
 * are overwritten.  `workspace` follows the rules of o1d_bwd_weight and
 * needs o1d_bwd_weight_workspace_bytes(...) bytes.  No output may overlap
 * an input, the other output or the workspace.  With N, H or W zero and
 * C > 0, dw is set to zeros. */
o1d_status_t o1d_bwd(const void* x, const void* dy, const void* w, const float* theta_deg, void* dx, void* dw,
                     int N, int C, int H, int W, int K, o1d_dtype_t dtype,
                     void* workspace, size_t workspace_bytes, void* stream);

/* Workspace size in bytes that o1d_bwd_weight (and o1d_bwd) needs for these sizes. */
size_t o1d_bwd_weight_workspace_bytes(int N, int C, int H, int W, int K, o1d_dtype_t dtype);

/* o1d_bwd without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation).  It computes exactly what o1d_bwd computes (the
 * same kernels and fixed-order sums, so dx and dw are bitwise equal to
 * o1d_bwd's) and keeps the weight gradient's partial rows in a fixed device scratch
 * array of 8 MiB that the library holds on every GPU it runs on until the
 * process ends.  It allocates and frees nothing.  Sizes whose partial rows
 * need more than 8 MiB (o1d_bwd_weight_workspace_bytes > 8 MiB) return
 * O1D_ERR_UNSUPPORTED before any launch.  All calls on one GPU share that
 * GPU's scratch: calls that overlap on one GPU (on different streams, or from
 * different threads without ordering) race and must be serialised by the
 * caller.  Nothing needs clearing between calls.  Other rules as o1d_bwd. */
o1d_status_t o1d_bwd_noalloc(const void* x, const void* dy, const void* w, const float* theta_deg, void* dx,
                             void* dw, int N, int C, int H, int W, int K, o1d_dtype_t dtype, void* stream);

/* ---- Stride, layout and sampling (Definition 1 with its stride `str`, Eq. 2).
 *
 * The _ex entry points compute the same three operations for any stride >= 1
 * (at most 64), either memory layout and either discretisation.  The input
 * plane is H x W; the output plane is P x Q with P = (H - 1) / stride + 1 and
 * Q = (W - 1) / stride + 1 (integer division: output (p, q) is centred on
 * input (stride p, stride q)):
 *   y[n,c,p,q]  = sum_k w[c,k] sample_k(x[n,c], stride p, stride q)
 *   dx[n,c,h,w] = the adjoint of that map in x (a scatter of dy, computed as a gather)
 *   dw[c,k]     = sum_{n,p,q} dy[n,c,p,q] sample_k(x[n,c], stride p, stride q)
 * where sample_k reads the pixel at the rounded-down offsets of Eq. (2)
 * (O1D_FLOOR) or interpolates bilinearly at the unrounded ones (O1D_BILINEAR),
 * pixels outside the plane reading zero.  Layouts: x and dx are N x C x H x W
 * (O1D_NCHW) or N x H x W x C (O1D_NHWC); y and dy are N x C x P x Q or
 * N x P x Q x C; w, dw are [C][K]; theta_deg is [C].  With stride 1, O1D_NCHW
 * and O1D_FLOOR they are exactly o1d_fwd, o1d_bwd_input and o1d_bwd_weight.
 * Ownership, asynchrony, precision, error and empty-tensor rules are those of
 * the plain entry points; H and W are always the input plane's, also for
 * o1d_bwd_input_ex.  O1D_ERR_UNSUPPORTED is returned where a band of the
 * plane with its zero margin does not fit in LDS (K and stride both very
 * large).  The weight gradient's workspace is
 * o1d_bwd_weight_ex_workspace_bytes(...) bytes. */
o1d_status_t o1d_fwd_ex(const void* x, const void* w, const float* theta_deg, void* y,
                        int N, int C, int H, int W, int K, int stride, o1d_layout_t layout,
                        o1d_sampling_t sampling, o1d_dtype_t dtype, void* stream);
o1d_status_t o1d_bwd_input_ex(const void* dy, const void* w, const float* theta_deg, void* dx,
                              int N, int C, int H, int W, int K, int stride, o1d_layout_t layout,
                              o1d_sampling_t sampling, o1d_dtype_t dtype, void* stream);
o1d_status_t o1d_bwd_weight_ex(const void* x, const void* dy, const float* theta_deg, void* dw,
                               int N, int C, int H, int W, int K, int stride, o1d_layout_t layout,
                               o1d_sampling_t sampling, o1d_dtype_t dtype,
                               void* workspace, size_t workspace_bytes, void* stream);
size_t o1d_bwd_weight_ex_workspace_bytes(int N, int C, int H, int W, int K, int stride, o1d_layout_t layout,
                                         o1d_sampling_t sampling, o1d_dtype_t dtype);

/* ---- Oriented 1D depthwise separable block (Sec. 3.2 "Computational cost
 * analysis", Table 1 "Oriented 1D DSC").
 *
 * The oriented depthwise convolution of Eq. (1) (stride 1, NCHW, offsets
 * rounded down) followed by a pointwise (1 x 1) convolution that mixes the C
 * channels into Cout:
 *   z = o1d_fwd(x, w_dw, theta_deg)                       (N x C x H x W)
 *   y[n,o,h,w] = sum_c w_pw[o,c] z[n,c,h,w]               (N x Cout x H x W)
 * w_dw is [C][K], w_pw [Cout][C] (row-major), theta_deg [C] float32; x, z, y,
 * w_dw and w_pw have `dtype` storage.  o1d_dsc_fwd writes z (kept for the
 * backward) and y; the pointwise product runs on the matrix cores (float32
 * products for O1D_F32, bfloat16 products for O1D_BF16, float32 accumulation).
 * o1d_dsc_bwd computes, for the upstream gradient dy (N x Cout x H x W):
 *   dz = w_pw^T dy (per pixel),  dw_pw[o,c] = sum_{n,h,w} dy[n,o,h,w] z[n,c,h,w],
 *   (dx, dw_dw) = o1d_bwd(x, dz, w_dw, theta_deg),
 * with dz kept in `workspace` (at least o1d_dsc_bwd_workspace_bytes(...)
 * bytes of caller-owned device memory, contents ignored and clobbered); its z
 * must be the forward's.  dw_pw's images are summed in groups whose float32
 * partial sums are added in a fixed order (bitwise reproducible).  Outputs
 * are overwritten; no output may overlap an input, another output or the
 * workspace.  Cout is 1 .. 65535; other rules as o1d_fwd and o1d_bwd. */
o1d_status_t o1d_dsc_fwd(const void* x, const void* w_dw, const float* theta_deg, const void* w_pw, void* z,
                         void* y, int N, int C, int Cout, int H, int W, int K, o1d_dtype_t dtype, void* stream);
o1d_status_t o1d_dsc_bwd(const void* x, const void* z, const void* dy, const void* w_dw, const float* theta_deg,
                         const void* w_pw, void* dx, void* dw_dw, void* dw_pw, int N, int C, int Cout, int H,
                         int W, int K, o1d_dtype_t dtype, void* workspace, size_t workspace_bytes, void* stream);
size_t o1d_dsc_bwd_workspace_bytes(int N, int C, int Cout, int H, int W, int K, o1d_dtype_t dtype);

/* ---- Planning introspection (host only, no device work; for tests and tools).
 *
 * o1d_kernel_name: the kernel(s) a call with these arguments would launch,
 * e.g. "strip_gather/f32/S77/KB32" or "gen_wgrad/bf16/nhwc/RP8/KB32"; two names
 * joined by '+' where o1d_bwd runs the input and weight gradients in turn.
 * op: 0 = o1d_fwd(_ex), 1 = o1d_bwd_input(_ex), 2 = o1d_bwd_weight(_ex),
 * 3 = o1d_bwd (stride 1, NCHW, O1D_FLOOR only).  `aligned` != 0 states that
 * the tensors are 16-byte (O1D_F32) or 8-byte (O1D_BF16) aligned.  Returns ""
 * for invalid or empty sizes.  The string lives in thread-local storage until
 * the thread's next call.
 * o1d_kernel_variant: the i-th kernel instantiation compiled into the
 * library, in the same naming, or NULL for i past the last. */
const char* o1d_kernel_name(int op, int N, int C, int H, int W, int K, int stride, o1d_layout_t layout,
                            o1d_sampling_t sampling, o1d_dtype_t dtype, int aligned);
const char* o1d_kernel_variant(int i);

/* Static description of a status code. */
const char* o1d_status_str(o1d_status_t status);

/* Detail for the calling thread's most recent non-OK status ("" if none). */
const char* o1d_last_error(void);

/* Library version string. */
const char* o1d_version(void);

#ifdef __cplusplus
}
#endif

#endif /* O1D_H_ */
