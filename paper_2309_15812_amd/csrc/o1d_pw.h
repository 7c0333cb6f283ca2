// Host-side plan of the pointwise (1 x 1) convolution of the oriented 1D
// depthwise separable block (Sec. 3.2, "Computational cost analysis", and
// Table 1's "Oriented 1D DSC"): a dense contraction over channels, run as a
// strided batched matrix product on the matrix cores.
//
//   C_b[m][n] = sum_k A_b[m][k] B_b[k][n]
//
// with element (m, k) of A_b at A + b sA + m am + k ak (strides in elements,
// likewise B and C).  The block's three products:
//   forward         Y_n  = Wp  Z_n   (M = C', N = H W, K = C, one batch per image)
//   input gradient  dZ_n = Wp^T dY_n (M = C,  N = H W, K = C')
//   weight gradient dWp  = sum_n dY_n Z_n^T (M = C', N = C, K = H W; the
//                   images are summed in nsplit groups whose float32
//                   partials are added in a fixed order)
#pragma once

#include <stddef.h>

#include "o1d_launch.h"
#include "o1d_plan.h"

namespace o1d {
namespace pw {

constexpr int kThreads = 256;  // four waves, 2 x 2 over the output tile
constexpr int kBM = 128, kBN = 128, kBK = 32;

struct Params {
  int M, N, K;
  int nbatch;                 // batches (images)
  long long sA, sB, sC;       // batch strides
  int am, ak, bk, bn, cm, cn;
  int a_kc, b_nc;             // A contiguous along k (else m), B contiguous along n (else k)
  int sum;                    // 1: batches are summed (nsplit groups of partials), 0: one output per batch
  int nsplit, per_split;      // summed: groups of per_split batches
  int tm, tn;                 // tiles along M and N
};

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

}  // namespace pw

// One translation unit per storage type; see o1d_pw_kernels.h.  `out` is
// the output tensor (sum == 0) or the float32 partials nsplit x M x N
// (sum == 1), which launch_pw_reduce then adds into the output.
#define O1D_PW_DECL(T)                                                                                          \
  hipError_t launch_pw_gemm_##T(const pw::Params& p, const void* A, const void* B, void* out, hipStream_t stream);
O1D_PW_DECL(f32)
O1D_PW_DECL(bf16)
#undef O1D_PW_DECL

inline hipError_t launch_pw_gemm(Dtype dt, const pw::Params& p, const void* A, const void* B, void* out,
                                 hipStream_t stream) {
  return dt == Dtype::F32 ? launch_pw_gemm_f32(p, A, B, out, stream) : launch_pw_gemm_bf16(p, A, B, out, stream);
}

}  // namespace o1d
