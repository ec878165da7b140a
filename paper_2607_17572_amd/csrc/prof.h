// Per-kernel-class launch timing with HIP events (measurement only).
//
// While a class is armed, prof_begin opens a record whose start and stop
// events are handed to the next launch made through jg::launch on the same
// host thread; that launch binds them to its own dispatch
// (hipExtLaunchKernelGGL), so the two timestamps are the kernel's start and
// end, not those of markers queued around it.
#pragma once
#include <hip/hip_ext.h>

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
// The record's events go to the next jg::launch of this thread.
int prof_begin(int cls);
// True while a kernel class is armed (the library then runs on one stream so
// that every timed kernel runs alone).
bool prof_armed();
// Closes record `idx` and attributes `work` (flops or bytes) to it; a record
// whose events no launch took (nothing was launched) is dropped.
void prof_end(int idx, double work);
// The pending record's events of this thread, consumed by the caller
// (false when there is none).
bool prof_take(hipEvent_t* start, hipEvent_t* stop);

// Kernel launch: plain when nothing is being timed, otherwise with the pending
// record's events bound to this dispatch.
template <typename F, typename... A>
inline void launch(F kern, dim3 grid, dim3 block, uint32_t lds, hipStream_t s, A... args) {
  hipEvent_t a = nullptr, b = nullptr;
  if (prof_armed() && prof_take(&a, &b))
    hipExtLaunchKernelGGL(kern, grid, block, lds, s, a, b, 0u, args...);
  else
    hipLaunchKernelGGL(kern, grid, block, lds, s, args...);
}

}  // namespace jg
