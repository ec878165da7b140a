// Per-kernel-class launch timing with HIP events (measurement only).
#pragma once
#include "common.h"

namespace jg {

enum ProfClass {
  PROF_NONE = 0,
  PROF_GEMM_FWD = 1,    // Y = X W^T
  PROF_GEMM_DGRAD = 2,  // dX = dY W
  PROF_GEMM_WGRAD = 3,  // dW = dY^T X
  PROF_ATTN_FWD = 4,
  PROF_ATTN_BWD_KV = 5,
  PROF_ATTN_BWD_Q = 6,
  PROF_AGGREGATE = 7,
  PROF_COMPARE = 8,     // gradient-quality sums
  PROF_UPSTREAM = 9,    // GRPO upstream gradients and their composites
};

// Returns a record index (>= 0) when class `cls` is being profiled, else -1.
int prof_begin(int cls, hipStream_t s);
// True while a kernel class is armed (the library then runs on one stream so
// that every timed kernel runs alone).
bool prof_armed();
// Closes record `idx` and attributes `work` (flops or bytes) to it.
void prof_end(int idx, hipStream_t s, double work);

}  // namespace jg
