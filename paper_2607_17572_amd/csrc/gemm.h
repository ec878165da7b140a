// GEMM entry of the JAGG HIP library.
//
//   C[m][n] (+)= epilogue( sum_k A(m,k) * B(n,k) )
//
// A(m,k) = ta ? A[k*lda + m] : A[m*lda + k]     (ta: A stored k-major, m contiguous)
// B(n,k) = tb ? B[k*ldb + n] : B[n*ldb + k]
//
// With weights stored [out][in], the three products of a linear layer are
//   forward   Y  = X W^T     ta=0, tb=0
//   input grad dX = dY W      ta=0, tb=1
//   weight grad dW = dY^T X   ta=1, tb=1   (contraction over token rows)
#pragma once
#include "common.h"

namespace jg {

enum EpiMode { EPI_STORE = 0, EPI_GELU_FWD = 1, EPI_GELU_BWD = 2 };

struct Epi {
  void* C = nullptr;
  int ldc = 0;
  int c_dt = F32;
  const void* bias = nullptr;  // per output column, added before the mode op
  int bias_dt = F32;
  float beta = 0.f;            // C = result + beta * C_old
  int mode = EPI_STORE;
  void* aux = nullptr;         // GELU_FWD: pre-activation out; GELU_BWD: pre-activation in
  int ldaux = 0;
  int aux_dt = BF16;
};

struct GemmArgs {
  const void* A = nullptr;
  int lda = 0, ta = 0, a_dt = BF16;
  const void* B = nullptr;
  int ldb = 0, tb = 0, b_dt = BF16;
  int M = 0, N = 0, K = 0;
  Epi epi;
};

// Returns 0 on success, 1 on invalid arguments, 3 on a launch error.
int gemm(const GemmArgs& g, hipStream_t s);

// Up to two independent products in one launch (for example the text- and
// image-stream products of one layer of a double-stream block): the problems
// keep their own operands, sizes and outputs; the tiles of the longer
// contraction come first.  Products the grouped kernel does not cover run as
// two gemm() calls.
struct GemmGroup {
  GemmArgs p[2];
  int np = 1;      // problems in the group
  int tiles0 = 0;  // workgroups of p[0] (set by the launcher)
};
int gemm2(const GemmArgs& a, const GemmArgs& b, hipStream_t s);

}  // namespace jg
