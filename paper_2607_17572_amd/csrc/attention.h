// Softmax attention forward/backward over the joint [text; image] sequence.
#pragma once
#include "ops.h"

namespace jg {

// Q, K, V: head-major [B][H][N][Dh] (act dtype).  O is written token-major
// into rows of the stream-major row layout (ld_o elements per row, head h at
// columns h*Dh ..), LSE [B][H][N] fp32 (natural log of sum exp of scaled scores).
struct AttnFwd {
  const void* Q; const void* K; const void* V;
  void* O; int ld_o;
  float* lse;
  int B, H, N, Dh, dt;
  RowMap rm;
};
int attention_fwd(const AttnFwd& a, hipStream_t s);

// dO token-major (ld_do), O token-major (ld_o); dQ/dK/dV head-major (dt_d).
// `delta` is workspace 2 x [B][H][N] fp32 (delta, then the log-sum-exp in
// log2 units for the MFMA kernels).
struct AttnBwd {
  const void* Q; const void* K; const void* V;
  const void* O; int ld_o;
  const void* dO; int ld_do;
  const float* lse;
  float* delta;
  void* dQ; void* dK; void* dV; int dt_d;
  int B, H, N, Dh, dt;
  RowMap rm;
  // bf16 MFMA path: the dK/dV kernel stores dS^T here and dQ = dS K is
  // formed from it without recomputing the scores (nullptr: the dQ kernel
  // recomputes them).  nk_pad x ld_ds elements per (sample, head), in chunks
  // of 128 keys x 64 queries (16 KB, key rows of 64 queries): element
  // (key k, query q) of head bh at
  //   ((bh * nk_pad / 128 + k / 128) * ld_ds / 64 + q / 64) * 8192
  //     + (k % 128) * 64 + q % 64,
  // so that one query tile of a key block is one contiguous 16 KB write and
  // the dQ pass streams contiguous 8 KB pieces.
  void* dS = nullptr;
  int ld_ds = 0, nk_pad = 0;
};
int attention_bwd(const AttnBwd& a, hipStream_t s);
// Padded dS^T geometry of the bf16 MFMA path: rows (keys) and columns
// (queries) to multiples of 128 (the key block of the dK/dV kernel and the
// query block of the dQ kernel).
inline int attn_ds_rows(int N) { return (N + 127) / 128 * 128; }
inline int attn_ds_ld(int N) { return (N + 127) / 128 * 128; }

}  // namespace jg
