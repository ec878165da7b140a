// Memory-bound kernels: adaLN / LayerNorm, gated residuals, q/k RMSNorm with
// 2-D rotary embedding, deterministic chunked column reductions, the small-M
// (batch) linear layers of the time MLP and modulation, and the JAGG
// aggregation and group-score kernels.  All arithmetic is fp32 (scores fp64);
// storage follows the activation dtype.
#include "ops.h"
#include "prof.h"

namespace jg {

#define LAUNCH_OK(name) JG_CHECK_LAUNCH(name)

__device__ inline int sample_of(const RowMap& rm, int r) {
  const int bt = rm.B * rm.nt;
  return r < bt ? r / rm.nt : (r - bt) / rm.ni;
}
__device__ inline bool is_txt(const RowMap& rm, int r) { return r < rm.B * rm.nt; }

// chunk q -> (first row, row count, sample)
__device__ inline void chunk_rows(const Chunks& c, int q, int& r0, int& n, int& b) {
  const int ct = c.ct(), ci = c.ci();
  if (q < c.B * ct) {
    b = q / ct;
    const int k = q % ct;
    r0 = b * c.nt + k * c.R;
    n = min(c.R, c.nt - k * c.R);
  } else {
    const int q2 = q - c.B * ct;
    b = q2 / ci;
    const int k = q2 % ci;
    r0 = c.B * c.nt + b * c.ni + k * c.R;
    n = min(c.R, c.ni - k * c.R);
  }
}

int chunk_range(RowMap rm, int row0, int nrows, int* c0, int* nc, int R) {
  Chunks c{rm.B, rm.nt, rm.ni, R};
  const int bt = rm.rows_txt();
  if (row0 == 0 && nrows == rm.rows()) { *c0 = 0; *nc = c.count(); return 0; }
  if (row0 == 0 && nrows == bt) { *c0 = 0; *nc = rm.B * c.ct(); return 0; }
  if (row0 == bt && nrows == rm.rows() - bt) { *c0 = rm.B * c.ct(); *nc = rm.B * c.ci(); return 0; }
  set_error("chunk_range: row range must be one stream or all rows");
  return 1;
}


// ---- vector helpers: 8 consecutive elements of a row ----
__device__ inline void ld8f(const uint16_t* p, float* f) {
  const uint4 u = *(const uint4*)p;
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) { f[2 * e] = bf2f(w[e] & 0xffffu); f[2 * e + 1] = bf2f(w[e] >> 16); }
}
__device__ inline void ld8f(const float* p, float* f) {
  const float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
  f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w; f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
}
// 8 consecutive elements of a row kept in their storage type (bf16: 4 VGPRs),
// converted to fp32 on use exactly as ld8f converts them
template <typename T>
struct Raw8;
template <>
struct Raw8<uint16_t> {
  uint4 u;
  __device__ inline void load(const uint16_t* p) { u = *(const uint4*)p; }
  __device__ inline float operator[](int e) const {
    const uint32_t w = e < 2 ? u.x : (e < 4 ? u.y : (e < 6 ? u.z : u.w));
    return bf2f((e & 1) ? (w >> 16) : (w & 0xffffu));
  }
};
template <>
struct Raw8<float> {
  float4 a, b;
  __device__ inline void load(const float* p) {
    a = *(const float4*)p;
    b = *(const float4*)(p + 4);
  }
  __device__ inline float operator[](int e) const {
    const float4 v = e < 4 ? a : b;
    const int k = e & 3;
    return k == 0 ? v.x : (k == 1 ? v.y : (k == 2 ? v.z : v.w));
  }
};
__device__ inline void st8f(uint16_t* p, const float* f) {
  uint4 u;
  u.x = f2bf(f[0]) | ((uint32_t)f2bf(f[1]) << 16);
  u.y = f2bf(f[2]) | ((uint32_t)f2bf(f[3]) << 16);
  u.z = f2bf(f[4]) | ((uint32_t)f2bf(f[5]) << 16);
  u.w = f2bf(f[6]) | ((uint32_t)f2bf(f[7]) << 16);
  *(uint4*)p = u;
}
__device__ inline void st8f(float* p, const float* f) {
  *(float4*)p = make_float4(f[0], f[1], f[2], f[3]);
  *(float4*)(p + 4) = make_float4(f[4], f[5], f[6], f[7]);
}
static inline bool al16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// ================================================================ small linear
template <typename TW>
__global__ __launch_bounds__(256) void small_linear_fwd_k(const float* __restrict__ in, int B, int Din,
                                                          const TW* __restrict__ W, const TW* __restrict__ bias,
                                                          float* __restrict__ out, int Dout) {
  const int lane = threadIdx.x & 63;
  const int j = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (j >= Dout) return;
  const TW* w = W + (size_t)j * Din;
  for (int b0 = 0; b0 < B; b0 += 8) {
    float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int d = lane; d < Din; d += 64) {
      const float wv = ldf(w, d);
#pragma unroll
      for (int bb = 0; bb < 8; ++bb)
        if (b0 + bb < B) acc[bb] = fmaf(wv, in[(size_t)(b0 + bb) * Din + d], acc[bb]);
    }
#pragma unroll
    for (int bb = 0; bb < 8; ++bb) {
      const float s = wave_sum(acc[bb]);
      if (lane == 0 && b0 + bb < B) out[(size_t)(b0 + bb) * Dout + j] = s + (bias ? ldf(bias, j) : 0.f);
    }
  }
}

// Wide rows (Din a multiple of 512): two output rows per wave, each lane
// reads 8 consecutive weights per 16-byte load (a wave streams 1 KB of W per
// instruction), the batch's inputs are read as 8-float vectors from cache.
template <typename TW>
__global__ __launch_bounds__(256) void small_linear_fwd_vec_k(const float* __restrict__ in, int B, int Din,
                                                              const TW* __restrict__ W, const TW* __restrict__ bias,
                                                              float* __restrict__ out, int Dout) {
  const int lane = threadIdx.x & 63;
  const int j0 = blockIdx.x * 8 + 2 * (threadIdx.x >> 6);
  if (j0 >= Dout) return;
  const bool two = j0 + 1 < Dout;
  const TW* w0 = W + (size_t)j0 * Din;
  const TW* w1 = W + (size_t)(two ? j0 + 1 : j0) * Din;
  for (int b0 = 0; b0 < B; b0 += 4) {
    float acc[2][4] = {{0, 0, 0, 0}, {0, 0, 0, 0}};
    for (int d = 8 * lane; d < Din; d += 512) {
      float a[8], c[8];
      ld8f(w0 + d, a);
      ld8f(w1 + d, c);
#pragma unroll
      for (int bb = 0; bb < 4; ++bb) {
        if (b0 + bb >= B) break;
        float x[8];
        ld8f(in + (size_t)(b0 + bb) * Din + d, x);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          acc[0][bb] = fmaf(a[e], x[e], acc[0][bb]);
          acc[1][bb] = fmaf(c[e], x[e], acc[1][bb]);
        }
      }
    }
#pragma unroll
    for (int bb = 0; bb < 4; ++bb) {
      const float s0 = wave_sum(acc[0][bb]), s1 = wave_sum(acc[1][bb]);
      if (lane == 0 && b0 + bb < B) {
        out[(size_t)(b0 + bb) * Dout + j0] = s0 + (bias ? ldf(bias, j0) : 0.f);
        if (two) out[(size_t)(b0 + bb) * Dout + j0 + 1] = s1 + (bias ? ldf(bias, j0 + 1) : 0.f);
      }
    }
  }
}

int small_linear_fwd(const float* in, int act, int B, int Din, const void* W, const void* bias, int w_dt,
                     float* out, int Dout, hipStream_t s) {
  if (act != 0 || B <= 0 || B > 64) { set_error("small_linear_fwd: bad batch/act"); return 1; }
  if (Din % 512 == 0 && al16(in) && al16(W)) {
    dim3 grid((Dout + 7) / 8);
    if (w_dt == BF16)
      hipLaunchKernelGGL(small_linear_fwd_vec_k<uint16_t>, grid, dim3(256), 0, s, in, B, Din, (const uint16_t*)W,
                         (const uint16_t*)bias, out, Dout);
    else
      hipLaunchKernelGGL(small_linear_fwd_vec_k<float>, grid, dim3(256), 0, s, in, B, Din, (const float*)W,
                         (const float*)bias, out, Dout);
    LAUNCH_OK("small_linear_fwd_vec");
    return 0;
  }
  dim3 grid((Dout + 3) / 4);
  if (w_dt == BF16)
    hipLaunchKernelGGL(small_linear_fwd_k<uint16_t>, grid, dim3(256), 0, s, in, B, Din, (const uint16_t*)W,
                       (const uint16_t*)bias, out, Dout);
  else
    hipLaunchKernelGGL(small_linear_fwd_k<float>, grid, dim3(256), 0, s, in, B, Din, (const float*)W,
                       (const float*)bias, out, Dout);
  LAUNCH_OK("small_linear_fwd");
  return 0;
}

constexpr int SL_JT = 64;   // output rows per tile
constexpr int SL_DT = 256;  // input columns per tile (one per thread)
constexpr int SL_MAXB = 32;

// Output rows per block of the vector kernel: enough blocks (~1024) to keep
// every CU streaming W and dW, at most SL_JT; the input-gradient partials
// grow with the block-row count.
static int sl_rows(int Din, int Dout) {
  const long cb = (Din + 1023) / 1024;
  const long r = cb * Dout / 1024 / 8 * 8;
  return (int)std::max<long>(8, std::min<long>(SL_JT, r));
}

size_t small_linear_bwd_part_floats(int B, int Din, int Dout) {
  const int jt = std::min(SL_JT, sl_rows(Din, Dout));
  return (size_t)((Dout + jt - 1) / jt) * B * Din;
}

template <typename TW, typename TG>
__global__ __launch_bounds__(256) void small_linear_bwd_k(const float* __restrict__ dout, const float* __restrict__ in,
                                                          int B, int Din, const TW* __restrict__ W, int Dout,
                                                          TG* __restrict__ dW, TG* __restrict__ db, float beta,
                                                          float* __restrict__ part) {
  __shared__ float sd[SL_MAXB][SL_JT];
  const int jt = blockIdx.y, j0 = jt * SL_JT;
  const int d = blockIdx.x * SL_DT + threadIdx.x;
  for (int i = threadIdx.x; i < B * SL_JT; i += 256) {
    const int b = i / SL_JT, jj = i % SL_JT;
    sd[b][jj] = (j0 + jj < Dout) ? dout[(size_t)b * Dout + j0 + jj] : 0.f;
  }
  __syncthreads();
  if (blockIdx.x == 0 && db) {
    for (int jj = threadIdx.x; jj < SL_JT; jj += 256) {
      if (j0 + jj >= Dout) continue;
      float s = 0.f;
      for (int b = 0; b < B; ++b) s += sd[b][jj];
      if (beta != 0.f) s += beta * ldf(db, j0 + jj);
      stf(db, j0 + jj, s);
    }
  }
  if (d >= Din) return;
  float x[SL_MAXB], acc[SL_MAXB];
  for (int b = 0; b < B; ++b) { x[b] = in[(size_t)b * Din + d]; acc[b] = 0.f; }
  const int jn = min(SL_JT, Dout - j0);
  // rows are independent apart from the input-gradient sums: unrolled so that
  // the loads of several rows are in flight together
#pragma unroll 8
  for (int jj = 0; jj < jn; ++jj) {
    const size_t idx = (size_t)(j0 + jj) * Din + d;
    const float w = ldf(W, idx);
    float g = 0.f;
    for (int b = 0; b < B; ++b) {
      g = fmaf(sd[b][jj], x[b], g);
      acc[b] = fmaf(sd[b][jj], w, acc[b]);
    }
    if (beta != 0.f) g += beta * ldf(dW, idx);
    stf(dW, idx, g);
  }
  if (part)
    for (int b = 0; b < B; ++b) part[((size_t)jt * B + b) * Din + d] = acc[b];
}

// out[i] (+)= sum over p of part[p * n + i], parts added in a fixed order: 64
// consecutive outputs per block, 4 slices of the parts per output (slice q
// sums parts q, q+4, ...), slices combined in order in LDS; acc: the sum is
// added to out's old value.
__global__ __launch_bounds__(256) void sum_parts_k(const float* __restrict__ part, int nparts, size_t n,
                                                   float* __restrict__ out, bool acc_out) {
  __shared__ float sl[4][64];
  const int c = threadIdx.x & 63, q = threadIdx.x >> 6;
  const size_t i = (size_t)blockIdx.x * 64 + c;
  float acc = 0.f;
  if (i < n) {
#pragma unroll 8
    for (int p = q; p < nparts; p += 4) acc += part[(size_t)p * n + i];
  }
  sl[q][c] = acc;
  __syncthreads();
  if (q == 0 && i < n) {
    const float t = ((sl[0][c] + sl[1][c]) + sl[2][c]) + sl[3][c];
    out[i] = acc_out ? out[i] + t : t;
  }
}

// Small batches: 8 consecutive input columns per thread (16-byte loads and
// stores of W and dW), all samples' rows kept in registers.
template <typename TW, typename TG, int BM>
__global__ __launch_bounds__(128) void small_linear_bwd_vec_k(const float* __restrict__ dout,
                                                              const float* __restrict__ in, int B, int Din,
                                                              const TW* __restrict__ W, int Dout, TG* __restrict__ dW,
                                                              TG* __restrict__ db, float beta,
                                                              float* __restrict__ part, int JT) {
  __shared__ float sd[BM][SL_JT];
  const int jt = blockIdx.y, j0 = jt * JT;
  for (int i = threadIdx.x; i < BM * JT; i += 128) {
    const int b = i / JT, jj = i % JT;
    sd[b][jj] = (b < B && j0 + jj < Dout) ? dout[(size_t)b * Dout + j0 + jj] : 0.f;
  }
  __syncthreads();
  if (blockIdx.x == 0 && db) {
    for (int jj = threadIdx.x; jj < JT; jj += 128) {
      if (j0 + jj >= Dout) continue;
      float sacc = 0.f;
      for (int b = 0; b < B; ++b) sacc += sd[b][jj];
      if (beta != 0.f) sacc += beta * ldf(db, j0 + jj);
      stf(db, j0 + jj, sacc);
    }
  }
  const int d = (blockIdx.x * 128 + threadIdx.x) * 8;
  if (d >= Din) return;
  float x[BM][8], acc[BM][8];
#pragma unroll
  for (int b = 0; b < BM; ++b) {
    if (b < B) ld8f(in + (size_t)b * Din + d, x[b]);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (b >= B) x[b][e] = 0.f;
      acc[b][e] = 0.f;
    }
  }
  const int jn = min(JT, Dout - j0);
  // rows are independent apart from the input-gradient sums: unrolled so that
  // the loads of several rows are in flight together
#pragma unroll 8
  for (int jj = 0; jj < jn; ++jj) {
    const size_t idx = (size_t)(j0 + jj) * Din + d;
    float w[8], gw[8];
    ld8f(W + idx, w);
#pragma unroll
    for (int e = 0; e < 8; ++e) gw[e] = 0.f;
#pragma unroll
    for (int b = 0; b < BM; ++b) {
      const float sv = sd[b][jj];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        gw[e] = fmaf(sv, x[b][e], gw[e]);
        acc[b][e] = fmaf(sv, w[e], acc[b][e]);
      }
    }
    if (beta != 0.f) {
      float o[8];
      ld8f(dW + idx, o);
#pragma unroll
      for (int e = 0; e < 8; ++e) gw[e] += beta * o[e];
    }
    st8f(dW + idx, gw);
  }
  if (part)
#pragma unroll
    for (int b = 0; b < BM; ++b)
      if (b < B) st8f(part + ((size_t)jt * B + b) * Din + d, acc[b]);
}

int small_linear_bwd(const float* dout, const float* in, int act, int B, int Din, const void* W, int w_dt,
                     int Dout, void* dW, void* db, int g_dt, float beta, float* din, float* part,
                     hipStream_t s, bool din_acc) {
  if (act != 0 || B <= 0 || B > SL_MAXB) { set_error("small_linear_bwd: batch must be 1..32"); return 1; }
  const int njt = (Dout + SL_JT - 1) / SL_JT;
  if (B <= 4 && Din % 8 == 0 && al16(in) && al16(W) && al16(dW) && (!din || al16(part))) {
    const int jt = sl_rows(Din, Dout), njv = (Dout + jt - 1) / jt;
    dim3 grid((Din + 1023) / 1024, njv);
    float* p = din ? part : nullptr;
#define SLV(TW, TG) \
  hipLaunchKernelGGL((small_linear_bwd_vec_k<TW, TG, 4>), grid, dim3(128), 0, s, dout, in, B, Din, (const TW*)W, Dout, \
                     (TG*)dW, (TG*)db, beta, p, jt)
    if (w_dt == BF16 && g_dt == BF16) SLV(uint16_t, uint16_t);
    else if (w_dt == BF16) SLV(uint16_t, float);
    else if (g_dt == BF16) SLV(float, uint16_t);
    else SLV(float, float);
#undef SLV
    LAUNCH_OK("small_linear_bwd_vec");
    if (din) {
      const size_t n = (size_t)B * Din;
      hipLaunchKernelGGL(sum_parts_k, dim3((n + 63) / 64), dim3(256), 0, s, part, njv, n, din, din_acc);
      LAUNCH_OK("small_linear_bwd_sum");
    }
    return 0;
  }
  dim3 grid((Din + SL_DT - 1) / SL_DT, njt);
  float* p = din ? part : nullptr;
#define SLB(TW, TG)                                                                                  \
  hipLaunchKernelGGL((small_linear_bwd_k<TW, TG>), grid, dim3(256), 0, s, dout, in, B, Din, (const TW*)W, \
                     Dout, (TG*)dW, (TG*)db, beta, p)
  if (w_dt == BF16 && g_dt == BF16) SLB(uint16_t, uint16_t);
  else if (w_dt == BF16) SLB(uint16_t, float);
  else if (g_dt == BF16) SLB(float, uint16_t);
  else SLB(float, float);
#undef SLB
  LAUNCH_OK("small_linear_bwd");
  if (din) {
    const size_t n = (size_t)B * Din;
    hipLaunchKernelGGL(sum_parts_k, dim3((n + 63) / 64), dim3(256), 0, s, part, njt, n, din, din_acc);
    LAUNCH_OK("small_linear_bwd_sum");
  }
  return 0;
}

// ================================================================ time embed
__global__ void time_embed_k(TVals tv, int B, int F, float* temb) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  const int half = F / 2;
  if (i >= B * half) return;
  const int b = i / half, k = i % half;
  // w_k = 10000^(-k/half); argument 1000 t w_k
  const double w = exp(-log(10000.0) * (double)k / (double)half);
  const double arg = 1000.0 * (double)tv.t[b] * w;
  temb[(size_t)b * F + k] = (float)cos(arg);
  temb[(size_t)b * F + half + k] = (float)sin(arg);
}

int time_embed(const TVals& tv, int B, int F, float* temb, hipStream_t s) {
  if (B <= 0 || B > 64 || F % 2) { set_error("time_embed: bad batch or width"); return 1; }
  const int n = B * F / 2;
  hipLaunchKernelGGL(time_embed_k, dim3((n + 255) / 256), dim3(256), 0, s, tv, B, F, temb);
  LAUNCH_OK("time_embed");
  return 0;
}

__global__ void silu_k(const float* x, float* y, size_t n) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) y[i] = silu(x[i]);
}
__global__ void mul_silu_grad_k(float* y, const float* x, size_t n) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) y[i] *= silu_grad(x[i]);
}
int silu_fwd(const float* x, float* y, size_t n, hipStream_t s) {
  hipLaunchKernelGGL(silu_k, dim3((n + 255) / 256), dim3(256), 0, s, x, y, n);
  LAUNCH_OK("silu");
  return 0;
}
int mul_silu_grad(float* y, const float* x, size_t n, hipStream_t s) {
  hipLaunchKernelGGL(mul_silu_grad_k, dim3((n + 255) / 256), dim3(256), 0, s, y, x, n);
  LAUNCH_OK("mul_silu_grad");
  return 0;
}

// ================================================================ LayerNorm + modulate
constexpr int MAXC = 16;  // columns per thread (D <= 4096 with 256 threads)

template <typename T>
__global__ __launch_bounds__(256) void ln_mod_fwd_k(const T* __restrict__ x, int D, RowMap rm, int row0,
                                                    const float* __restrict__ mt, const float* __restrict__ mi,
                                                    int mod_w, int sh_off, int sc_off, T* __restrict__ a,
                                                    float* __restrict__ mean, float* __restrict__ rstd) {
  __shared__ float sh[16];
  const int r = row0 + blockIdx.x;
  const T* xr = x + (size_t)r * D;
  float v[MAXC];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = threadIdx.x + i * 256;
    v[i] = c < D ? ldf(xr, c) : 0.f;
    s += v[i];
  }
  const float mu = block_sum(s, sh) / D;
  float s2 = 0.f;
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = threadIdx.x + i * 256;
    const float dlt = c < D ? v[i] - mu : 0.f;
    s2 += dlt * dlt;
  }
  const float var = block_sum(s2, sh) / D;
  const float rs = rsqrtf(var + 1e-6f);
  const int b = sample_of(rm, r);
  const float* m = (is_txt(rm, r) ? mt : mi) + (size_t)b * mod_w;
  T* ar = a + (size_t)r * D;
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = threadIdx.x + i * 256;
    if (c < D) stf(ar, c, (v[i] - mu) * rs * (1.f + m[sc_off + c]) + m[sh_off + c]);
  }
  if (threadIdx.x == 0) { mean[r] = mu; rstd[r] = rs; }
}

// Hidden sizes that are multiples of 512: one wave per row, 8 consecutive
// columns per lane and access (lane columns 8 lane + 512 i), the row's mean
// and variance from wave reductions.
template <typename T, int NV>
__global__ __launch_bounds__(256) void ln_mod_fwd_vec_k(const T* __restrict__ x, RowMap rm, int row0, int nrows,
                                                        const float* __restrict__ mt, const float* __restrict__ mi,
                                                        int mod_w, int sh_off, int sc_off, T* __restrict__ a,
                                                        float* __restrict__ mean, float* __restrict__ rstd) {
  constexpr int D = NV * 512;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int rr = blockIdx.x * 4 + w;
  if (rr >= nrows) return;
  const int r = row0 + rr;
  float v[NV * 8];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) ld8f(x + (size_t)r * D + 8 * lane + 512 * i, v + 8 * i);
#pragma unroll
  for (int e = 0; e < NV * 8; ++e) s += v[e];
  const float mu = wave_sum(s) / D;
  float s2 = 0.f;
#pragma unroll
  for (int e = 0; e < NV * 8; ++e) {
    const float dlt = v[e] - mu;
    s2 += dlt * dlt;
  }
  const float var = wave_sum(s2) / D;
  const float rs = rsqrtf(var + 1e-6f);
  const float* m = (is_txt(rm, r) ? mt : mi) + (size_t)sample_of(rm, r) * mod_w;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = 8 * lane + 512 * i;
    float sc[8], sf[8], o[8];
    ld8f(m + sc_off + c, sc);
    ld8f(m + sh_off + c, sf);
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = (v[8 * i + e] - mu) * rs * (1.f + sc[e]) + sf[e];
    st8f(a + (size_t)r * D + c, o);
  }
  if (lane == 0) {
    mean[r] = mu;
    rstd[r] = rs;
  }
}

int ln_mod_fwd(const void* x, int act_dt, int D, RowMap rm, int row0, int nrows, const float* mod_txt,
               const float* mod_img, int mod_w, int sh_off, int sc_off, void* a, float* mean, float* rstd,
               hipStream_t s) {
  if (D > 256 * MAXC) { set_error("ln_mod_fwd: hidden too large"); return 1; }
  if (nrows <= 0) return 0;
  if (D % 512 == 0 && D <= 3584 && al16(x) && al16(a) && al16(mod_txt) && al16(mod_img) && mod_w % 4 == 0 &&
      sh_off % 4 == 0 && sc_off % 4 == 0) {
    const dim3 grid((unsigned)((nrows + 3) / 4));
#define LNF(T, NV)                                                                                                \
  case NV:                                                                                                        \
    hipLaunchKernelGGL((ln_mod_fwd_vec_k<T, NV>), grid, dim3(256), 0, s, (const T*)x, rm, row0, nrows, mod_txt,  \
                       mod_img, mod_w, sh_off, sc_off, (T*)a, mean, rstd);                                       \
    break;
    if (act_dt == BF16) {
      switch (D / 512) { LNF(uint16_t, 1) LNF(uint16_t, 2) LNF(uint16_t, 3) LNF(uint16_t, 4) LNF(uint16_t, 5)
                         LNF(uint16_t, 6) LNF(uint16_t, 7) }
    } else {
      switch (D / 512) { LNF(float, 1) LNF(float, 2) LNF(float, 3) LNF(float, 4) LNF(float, 5) LNF(float, 6)
                         LNF(float, 7) }
    }
#undef LNF
    LAUNCH_OK("ln_mod_fwd_vec");
    return 0;
  }
  if (act_dt == BF16)
    hipLaunchKernelGGL(ln_mod_fwd_k<uint16_t>, dim3(nrows), dim3(256), 0, s, (const uint16_t*)x, D, rm, row0,
                       mod_txt, mod_img, mod_w, sh_off, sc_off, (uint16_t*)a, mean, rstd);
  else
    hipLaunchKernelGGL(ln_mod_fwd_k<float>, dim3(nrows), dim3(256), 0, s, (const float*)x, D, rm, row0, mod_txt,
                       mod_img, mod_w, sh_off, sc_off, (float*)a, mean, rstd);
  LAUNCH_OK("ln_mod_fwd");
  return 0;
}

template <typename T, typename TG>
__global__ __launch_bounds__(256) void ln_mod_bwd_k(const float* __restrict__ dA, const T* __restrict__ x, int D,
                                                    Chunks ch, int c0, const float* __restrict__ mean,
                                                    const float* __restrict__ rstd, const float* __restrict__ mt,
                                                    const float* __restrict__ mi, int mod_w, int sc_off,
                                                    const TG* gin, float* g, float* __restrict__ psc,
                                                    float* __restrict__ psh) {
  __shared__ float sh[16];
  const int q = c0 + blockIdx.x;
  int r0, n, b;
  chunk_rows(ch, q, r0, n, b);
  const bool txt = r0 < ch.B * ch.nt;
  const float* m = (txt ? mt : mi) + (size_t)b * mod_w + sc_off;
  float scl[MAXC], asc[MAXC], ash[MAXC];
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = threadIdx.x + i * 256;
    scl[i] = c < D ? 1.f + m[c] : 0.f;
    asc[i] = 0.f;
    ash[i] = 0.f;
  }
  for (int rr = 0; rr < n; ++rr) {
    const int r = r0 + rr;
    const float mu = mean[r], rs = rstd[r];
    float xh[MAXC], dxh[MAXC];
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
      const int c = threadIdx.x + i * 256;
      if (c < D) {
        const float da = dA[(size_t)r * D + c];
        xh[i] = (ldf(x, (size_t)r * D + c) - mu) * rs;
        dxh[i] = da * scl[i];
        asc[i] = fmaf(da, xh[i], asc[i]);
        ash[i] += da;
        s1 += dxh[i];
        s2 += dxh[i] * xh[i];
      } else {
        xh[i] = dxh[i] = 0.f;
      }
    }
    const float m1 = block_sum(s1, sh) / D;
    const float m2 = block_sum(s2, sh) / D;
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
      const int c = threadIdx.x + i * 256;
      if (c < D) g[(size_t)r * D + c] = ldf(gin, (size_t)r * D + c) + rs * (dxh[i] - m1 - xh[i] * m2);
    }
  }
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = threadIdx.x + i * 256;
    if (c < D) {
      psc[(size_t)q * D + c] = asc[i];
      psh[(size_t)q * D + c] = ash[i];
    }
  }
}

// One wave per row (rows of the chunk dealt round-robin to the LN_W waves),
// each lane owning NV runs of 8 consecutive columns (16-byte loads).  The
// per-sample factors 1 + scale sit in LDS, x stays in its storage type and the
// shift-gradient column sums accumulate in the wave's own LDS row, so a wave
// keeps under 256 VGPRs and two blocks share a CU.  A block takes LN_ROWS
// rows, so the many blocks spread evenly over the CUs.  The per-column partial
// sums of the waves are combined through LDS in wave order.
constexpr int LN_W = 4;
template <typename T, typename TG, int NV>
__global__ __launch_bounds__(64 * LN_W) __attribute__((amdgpu_waves_per_eu(2, 2))) void ln_mod_bwd_vec_k(
    const float* __restrict__ dA, const T* __restrict__ x, Chunks ch, int c0, const float* __restrict__ mean,
    const float* __restrict__ rstd, const float* __restrict__ mt, const float* __restrict__ mi, int mod_w,
    int sc_off, const TG* gin, float* g, float* __restrict__ psc, float* __restrict__ psh) {
  constexpr int D = NV * 512;
  extern __shared__ float red[];  // [LN_W][D] column sums per wave, then [D] factors 1 + scale
  float* const ms = red + LN_W * D;
  const int q = c0 + blockIdx.x;
  int r0, n, b;
  chunk_rows(ch, q, r0, n, b);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const float* mg = ((r0 < ch.B * ch.nt) ? mt : mi) + (size_t)b * mod_w + sc_off;
  for (int c = threadIdx.x; c < D; c += 64 * LN_W) ms[c] = mg[c] + 1.f;
  float* const sh = red + w * D + 8 * lane;  // this lane's shift sums
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    *(float4*)(sh + 512 * i) = make_float4(0.f, 0.f, 0.f, 0.f);
    *(float4*)(sh + 512 * i + 4) = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  __syncthreads();
  float asc[NV * 8];
#pragma unroll
  for (int i = 0; i < NV * 8; ++i) asc[i] = 0.f;
  Raw8<T> xr[NV];
  float da[NV * 8];
  for (int rr = w; rr < n; rr += LN_W) {
    const int r = r0 + rr;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      xr[i].load(x + (size_t)r * D + 8 * lane + 512 * i);
      ld8f(dA + (size_t)r * D + 8 * lane + 512 * i, da + 8 * i);
    }
    const float mu = mean[r], rs = rstd[r];
    // opaque per row: the factor reads stay in the loop instead of being
    // hoisted into 48 registers
    int mo = 8 * lane;
    asm volatile("" : "+v"(mo));
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      float m[8], t[8];
      ld8f(ms + mo + 512 * i, m);
      ld8f(sh + 512 * i, t);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int k = 8 * i + e;
        const float xhat = (xr[i][e] - mu) * rs;
        const float d = da[k] * m[e];
        asc[k] = fmaf(da[k], xhat, asc[k]);
        t[e] += da[k];
        s1 += d;
        s2 += d * xhat;
      }
      st8f(sh + 512 * i, t);
    }
    const float m1 = wave_sum(s1) / D, m2 = wave_sum(s2) / D;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int c = 8 * lane + 512 * i;
      float m[8], gv[8];
      ld8f(ms + mo + 512 * i, m);
      ld8f(gin + (size_t)r * D + c, gv);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float xhat = (xr[i][e] - mu) * rs;
        gv[e] += rs * (da[8 * i + e] * m[e] - m1 - xhat * m2);
      }
      st8f(g + (size_t)r * D + c, gv);
      // one 8-column block at a time: hoisting all gradient loads spills
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  // shift sums first (already in LDS), then the scale sums through the same rows
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    if (pass == 1) {
#pragma unroll
      for (int i = 0; i < NV; ++i) st8f(sh + 512 * i, asc + 8 * i);
    }
    __syncthreads();
    float* out = (pass == 0 ? psh : psc) + (size_t)q * D;
    for (int c = threadIdx.x; c < D; c += 64 * LN_W) {
      float t = red[c];
#pragma unroll
      for (int k = 1; k < LN_W; ++k) t += red[k * D + c];
      out[c] = t;
    }
    __syncthreads();
  }
}

int ln_mod_bwd(const float* dA, const void* x, int act_dt, int D, RowMap rm, int row0, int nrows,
               const float* mean, const float* rstd, const float* mod_txt, const float* mod_img, int mod_w,
               int sc_off, const void* g_in, int g_in_dt, float* g, float* part_scale, float* part_shift,
               hipStream_t s) {
  if (D > 256 * MAXC) { set_error("ln_mod_bwd: hidden too large"); return 1; }
  if (g_in_dt == BF16 && act_dt != BF16) {
    set_error("ln_mod_bwd: a bf16 incoming gradient needs bf16 activations");
    return 1;
  }
  int c0, nc;
  if (chunk_range(rm, row0, nrows, &c0, &nc, LN_ROWS)) return 1;
  if (nc == 0) return 0;
  Chunks ch{rm.B, rm.nt, rm.ni, LN_ROWS};
  if (D % 512 == 0 && D <= 3584 && al16(dA) && al16(x) && al16(g) && al16(g_in)) {
    const size_t lds = (LN_W + 1) * (size_t)D * sizeof(float);
#define LNB(T, TG, NV)                                                                                         \
  case NV: {                                                                                                   \
    auto k = ln_mod_bwd_vec_k<T, TG, NV>;                                                                      \
    if (lds > 65536 &&                                                                                         \
        hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess) { \
      set_error("ln_mod_bwd: cannot reserve the row buffers in LDS");                                          \
      return 3;                                                                                                \
    }                                                                                                          \
    hipLaunchKernelGGL(k, dim3(nc), dim3(64 * LN_W), lds, s, dA, (const T*)x, ch, c0, mean, rstd, mod_txt, mod_img, \
                       mod_w, sc_off, (const TG*)g_in, g, part_scale, part_shift);                              \
  } break;
#define LNS(T, TG) \
  switch (D / 512) { LNB(T, TG, 1) LNB(T, TG, 2) LNB(T, TG, 3) LNB(T, TG, 4) LNB(T, TG, 5) LNB(T, TG, 6) LNB(T, TG, 7) }
    if (act_dt == BF16 && g_in_dt == BF16) LNS(uint16_t, uint16_t)
    else if (act_dt == BF16) LNS(uint16_t, float)
    else LNS(float, float)
#undef LNS
#undef LNB
    LAUNCH_OK("ln_mod_bwd_vec");
    return 0;
  }
#define LNK(T, TG)                                                                                              \
  hipLaunchKernelGGL((ln_mod_bwd_k<T, TG>), dim3(nc), dim3(256), 0, s, dA, (const T*)x, D, ch, c0, mean, rstd, \
                     mod_txt, mod_img, mod_w, sc_off, (const TG*)g_in, g, part_scale, part_shift)
  if (act_dt == BF16 && g_in_dt == BF16) LNK(uint16_t, uint16_t);
  else if (act_dt == BF16) LNK(uint16_t, float);
  else LNK(float, float);
#undef LNK
  LAUNCH_OK("ln_mod_bwd");
  return 0;
}

// ================================================================ gated residual
template <typename T>
__global__ void gated_residual_k(const T* __restrict__ xi, const T* __restrict__ y, int D, int ld_y, RowMap rm,
                                 int row0, size_t n, const float* __restrict__ mt, const float* __restrict__ mi,
                                 int mod_w, int gate_off, T* __restrict__ xo) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int r = row0 + (int)(i / D), c = (int)(i % D);
  const int b = sample_of(rm, r);
  const float gt = ((is_txt(rm, r) ? mt : mi) + (size_t)b * mod_w)[gate_off + c];
  const size_t xidx = (size_t)r * D + c;
  stf(xo, xidx, ldf(xi, xidx) + gt * ldf(y, (size_t)r * ld_y + c));
}

// 8 consecutive columns of one row per thread (D a multiple of 8): 16-byte
// accesses, the same arithmetic per element as gated_residual_k
template <typename T>
__global__ void gated_residual8_k(const T* __restrict__ xi, const T* __restrict__ y, int D, int ld_y, RowMap rm,
                                  int row0, size_t n8, const float* __restrict__ mt, const float* __restrict__ mi,
                                  int mod_w, int gate_off, T* __restrict__ xo) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n8) return;
  const size_t e0 = 8 * i;
  const int r = row0 + (int)(e0 / D), c = (int)(e0 % D);
  const float* gp = (is_txt(rm, r) ? mt : mi) + (size_t)sample_of(rm, r) * mod_w + gate_off + c;
  float xv[8], yv[8], gt[8], o[8];
  ld8f(xi + (size_t)r * D + c, xv);
  ld8f(y + (size_t)r * ld_y + c, yv);
  ld8f(gp, gt);
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = xv[e] + gt[e] * yv[e];
  st8f(xo + (size_t)r * D + c, o);
}

int gated_residual(const void* xi, const void* y, int act_dt, int D, int ld_y, RowMap rm, int row0, int nrows,
                   const float* mod_txt, const float* mod_img, int mod_w, int gate_off, void* xo,
                   hipStream_t s) {
  const size_t n = (size_t)nrows * D;
  if (n == 0) return 0;
  if (D % 8 == 0 && ld_y % 8 == 0 && al16(xi) && al16(y) && al16(xo) && al16(mod_txt) && al16(mod_img) &&
      mod_w % 4 == 0 && gate_off % 4 == 0) {
    const size_t n8 = n / 8;
    const dim3 grid((unsigned)((n8 + 255) / 256));
    if (act_dt == BF16)
      hipLaunchKernelGGL(gated_residual8_k<uint16_t>, grid, dim3(256), 0, s, (const uint16_t*)xi,
                         (const uint16_t*)y, D, ld_y, rm, row0, n8, mod_txt, mod_img, mod_w, gate_off, (uint16_t*)xo);
    else
      hipLaunchKernelGGL(gated_residual8_k<float>, grid, dim3(256), 0, s, (const float*)xi, (const float*)y, D, ld_y,
                         rm, row0, n8, mod_txt, mod_img, mod_w, gate_off, (float*)xo);
    LAUNCH_OK("gated_residual");
    return 0;
  }
  dim3 grid((unsigned)((n + 255) / 256));
  if (act_dt == BF16)
    hipLaunchKernelGGL(gated_residual_k<uint16_t>, grid, dim3(256), 0, s, (const uint16_t*)xi, (const uint16_t*)y,
                       D, ld_y, rm, row0, n, mod_txt, mod_img, mod_w, gate_off, (uint16_t*)xo);
  else
    hipLaunchKernelGGL(gated_residual_k<float>, grid, dim3(256), 0, s, (const float*)xi, (const float*)y, D, ld_y,
                       rm, row0, n, mod_txt, mod_img, mod_w, gate_off, (float*)xo);
  LAUNCH_OK("gated_residual");
  return 0;
}

template <typename T, typename TG>
__global__ __launch_bounds__(256) void gate_bwd_k(const TG* __restrict__ g, const T* __restrict__ y, int D,
                                                  Chunks ch, int c0, const float* __restrict__ mt,
                                                  const float* __restrict__ mi, int mod_w, int gate_off,
                                                  T* __restrict__ dY, int ld_dy, float* __restrict__ pg,
                                                  float* __restrict__ pb) {
  const int q = c0 + blockIdx.x;
  int r0, n, b;
  chunk_rows(ch, q, r0, n, b);
  const float* m = ((r0 < ch.B * ch.nt) ? mt : mi) + (size_t)b * mod_w + gate_off;
  for (int c = threadIdx.x; c < D; c += 256) {
    const float gt = m[c];
    float sg = 0.f, sb = 0.f;
    for (int rr = 0; rr < n; ++rr) {
      const int r = r0 + rr;
      const float gv = ldf(g, (size_t)r * D + c);
      sg = fmaf(gv, ldf(y, (size_t)r * D + c), sg);
      const float d = gv * gt;
      sb += d;
      stf(dY, (size_t)r * ld_dy + c, d);
    }
    pg[(size_t)q * D + c] = sg;
    pb[(size_t)q * D + c] = sb;
  }
}

// At most 4 waves per SIMD, so that the compiler may keep four rows' loads in
// registers (at 8 waves it reused the load registers and waited per load).
template <typename T, typename TG>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 4))) void gate_bwd_vec_k(
    const TG* __restrict__ g, const T* __restrict__ y, int D, Chunks ch, int c0, const float* __restrict__ mt,
    const float* __restrict__ mi, int mod_w, int gate_off, T* __restrict__ dY, int ld_dy, float* __restrict__ pg,
    float* __restrict__ pb) {
  const int q = c0 + blockIdx.x;
  int r0, n, b;
  chunk_rows(ch, q, r0, n, b);
  const int c = (blockIdx.y * 256 + threadIdx.x) * 8;
  if (c >= D) return;
  const float* m = ((r0 < ch.B * ch.nt) ? mt : mi) + (size_t)b * mod_w + gate_off + c;
  float gt[8], sg[8], sb[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) { gt[e] = m[e]; sg[e] = 0.f; sb[e] = 0.f; }
  auto row = [&](const Raw8<TG>& gv, const Raw8<T>& yv, int r) {
    float d[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      sg[e] = fmaf(gv[e], yv[e], sg[e]);
      d[e] = gv[e] * gt[e];
      sb[e] += d[e];
    }
    st8f(dY + (size_t)r * ld_dy + c, d);
  };
  // four rows' loads issued together, then the rows in order
  int rr = 0;
  for (; rr + 4 <= n; rr += 4) {
    Raw8<TG> gv[4];
    Raw8<T> yv[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      gv[k].load(g + (size_t)(r0 + rr + k) * D + c);
      yv[k].load(y + (size_t)(r0 + rr + k) * D + c);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) row(gv[k], yv[k], r0 + rr + k);
  }
  for (; rr < n; ++rr) {
    Raw8<TG> gv;
    Raw8<T> yv;
    gv.load(g + (size_t)(r0 + rr) * D + c);
    yv.load(y + (size_t)(r0 + rr) * D + c);
    row(gv, yv, r0 + rr);
  }
  st8f(pg + (size_t)q * D + c, sg);
  st8f(pb + (size_t)q * D + c, sb);
}

int gate_bwd(const void* g, int g_dt, const void* y, int act_dt, int D, RowMap rm, int row0, int nrows,
             const float* mod_txt, const float* mod_img, int mod_w, int gate_off, void* dY, int ld_dy,
             float* part_gate, float* part_bias, hipStream_t s) {
  if (g_dt == BF16 && act_dt != BF16) {
    set_error("gate_bwd: a bf16 incoming gradient needs bf16 activations");
    return 1;
  }
  int c0, nc;
  if (chunk_range(rm, row0, nrows, &c0, &nc)) return 1;
  if (nc == 0) return 0;
  Chunks ch{rm.B, rm.nt, rm.ni, RED_ROWS};
  if (D % 8 == 0 && ld_dy % 8 == 0 && mod_w % 4 == 0 && gate_off % 4 == 0 && al16(g) && al16(y) && al16(dY) &&
      al16(mod_txt) && al16(mod_img) && al16(part_gate) && al16(part_bias)) {
    dim3 grid(nc, (D + 2047) / 2048);
#define GBV(T, TG)                                                                                             \
  hipLaunchKernelGGL((gate_bwd_vec_k<T, TG>), grid, dim3(256), 0, s, (const TG*)g, (const T*)y, D, ch, c0, mod_txt, \
                     mod_img, mod_w, gate_off, (T*)dY, ld_dy, part_gate, part_bias)
    if (act_dt == BF16 && g_dt == BF16) GBV(uint16_t, uint16_t);
    else if (act_dt == BF16) GBV(uint16_t, float);
    else GBV(float, float);
#undef GBV
    LAUNCH_OK("gate_bwd_vec");
    return 0;
  }
#define GBK(T, TG)                                                                                              \
  hipLaunchKernelGGL((gate_bwd_k<T, TG>), dim3(nc), dim3(256), 0, s, (const TG*)g, (const T*)y, D, ch, c0, mod_txt, \
                     mod_img, mod_w, gate_off, (T*)dY, ld_dy, part_gate, part_bias)
  if (act_dt == BF16 && g_dt == BF16) GBK(uint16_t, uint16_t);
  else if (act_dt == BF16) GBK(uint16_t, float);
  else GBK(float, float);
#undef GBK
  LAUNCH_OK("gate_bwd");
  return 0;
}

// ================================================================ q/k norm + rope
__device__ inline void tok_of_row(const RowMap& rm, int r, int& b, int& j) {
  const int bt = rm.B * rm.nt;
  if (r < bt) { b = r / rm.nt; j = r % rm.nt; }
  else { b = (r - bt) / rm.ni; j = rm.nt + (r - bt) % rm.ni; }
}

// angle of rotation pair p for joint token j
__device__ inline float rope_angle(const Rope& rp, int j, int p) {
  float pos = 0.f;
  const int quarter = rp.Dh / 4;
  if (j >= rp.nt) {
    const int i = j - rp.nt;
    pos = (p < quarter) ? (float)(i / rp.gw) : (float)(i % rp.gw);
  }
  const int k = p % quarter;
  const float freq = exp2f(-(2.f * k / (rp.Dh / 2)) * 13.287712379549449f);  // log2(1e4)
  return pos * freq;
}

template <typename T>
__global__ __launch_bounds__(256) void qk_norm_rope_fwd_k(const T* __restrict__ proj, int ld, RowMap rm, Rope rp,
                                                          Gains gn, T* __restrict__ Qh, T* __restrict__ Kh,
                                                          T* __restrict__ Vh, float* __restrict__ rq,
                                                          float* __restrict__ rk, int nitems) {
  const int item = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (item >= nitems) return;
  const int lane = threadIdx.x & 63;
  const int r = item / rp.H, h = item % rp.H;
  const int D = rp.H * rp.Dh;
  const bool act = lane < rp.Dh / 2;
  const int p = act ? lane : 0;
  const T* pr = proj + (size_t)r * ld;
  const int st = r < rm.B * rm.nt ? 0 : 1;
  const T* qg = (const T*)gn.q[st];
  const T* kg = (const T*)gn.k[st];
  float q0 = 0, q1 = 0, k0 = 0, k1 = 0;
  if (act) {
    q0 = ldf(pr, h * rp.Dh + 2 * p);
    q1 = ldf(pr, h * rp.Dh + 2 * p + 1);
    k0 = ldf(pr, D + h * rp.Dh + 2 * p);
    k1 = ldf(pr, D + h * rp.Dh + 2 * p + 1);
  }
  const float riq = rsqrtf(wave_sum(q0 * q0 + q1 * q1) / rp.Dh + 1e-6f);
  const float rik = rsqrtf(wave_sum(k0 * k0 + k1 * k1) / rp.Dh + 1e-6f);
  if (lane == 0) { rq[(size_t)r * rp.H + h] = riq; rk[(size_t)r * rp.H + h] = rik; }
  if (!act) return;
  int b, j;
  tok_of_row(rm, r, b, j);
  const int N = rm.nt + rm.ni;
  float sn, cs;
  sincosf(rope_angle(rp, j, p), &sn, &cs);
  const float qa = q0 * riq * ldf(qg, 2 * p), qb = q1 * riq * ldf(qg, 2 * p + 1);
  const float ka = k0 * rik * ldf(kg, 2 * p), kb = k1 * rik * ldf(kg, 2 * p + 1);
  const size_t o = (((size_t)b * rp.H + h) * N + j) * rp.Dh + 2 * p;
  stf(Qh, o, qa * cs - qb * sn);
  stf(Qh, o + 1, qa * sn + qb * cs);
  stf(Kh, o, ka * cs - kb * sn);
  stf(Kh, o + 1, ka * sn + kb * cs);
  stf(Vh, o, ldf(pr, 2 * D + h * rp.Dh + 2 * p));
  stf(Vh, o + 1, ldf(pr, 2 * D + h * rp.Dh + 2 * p + 1));
}

template <typename T>
__global__ void qk_norm_rope_fwd_row_k(const T* __restrict__ proj, int ld, RowMap rm, Rope rp, Gains gn,
                                       T* __restrict__ Qh, T* __restrict__ Kh, T* __restrict__ Vh,
                                       float* __restrict__ rq, float* __restrict__ rk);

// Forward for bf16 and head_dim 128 with 16-byte accesses, one wave per row:
// per step the wave takes four heads, 16 lanes per head, each lane 4 RoPE
// pairs (8 consecutive elements).  The rotation of pair p is computed once per
// row by lane p and handed to the lanes that use it; the RMS sums run over the
// 16 lanes of a head.
__global__ __launch_bounds__(256) void qk_norm_rope_fwd8_k(const uint16_t* __restrict__ proj, int ld, RowMap rm,
                                                           Rope rp, Gains gn, uint16_t* __restrict__ Qh,
                                                           uint16_t* __restrict__ Kh, uint16_t* __restrict__ Vh,
                                                           float* __restrict__ rq, float* __restrict__ rk) {
  constexpr int Dh = 128;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rm.rows()) return;
  const int lane = threadIdx.x & 63, hq = lane >> 4, lp = lane & 15, e0 = 8 * lp;
  const int H = rp.H, D = H * Dh, N = rm.nt + rm.ni;
  const int st = r < rm.B * rm.nt ? 0 : 1;
  float qg[8], kg[8];
  ld8f((const uint16_t*)gn.q[st] + e0, qg);
  ld8f((const uint16_t*)gn.k[st] + e0, kg);
  int b, j;
  tok_of_row(rm, r, b, j);
  float sn0, cs0;
  sincosf(rope_angle(rp, j, lane), &sn0, &cs0);
  float cs[4], sn[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    cs[k] = __shfl(cs0, 4 * lp + k, 64);
    sn[k] = __shfl(sn0, 4 * lp + k, 64);
  }
  const uint16_t* pr = proj + (size_t)r * ld + e0;
  const size_t ob = ((size_t)b * H * N + j) * Dh + e0;  // head h adds h * N * Dh
  for (int h0 = 0; h0 < H; h0 += 4) {
    const int h = h0 + hq;
    const bool hv = h < H;
    const int hh = hv ? h : 0;  // lanes past the last head compute on head 0, store nothing
    float x[8], y[8];
    ld8f(pr + hh * Dh, x);
    ld8f(pr + D + hh * Dh, y);
    const uint4 vv = *(const uint4*)(pr + 2 * D + hh * Dh);
    float sq = 0.f, sk = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      sq = fmaf(x[e], x[e], sq);
      sk = fmaf(y[e], y[e], sk);
    }
#pragma unroll
    for (int m = 8; m > 0; m >>= 1) {
      sq += __shfl_xor(sq, m, 16);
      sk += __shfl_xor(sk, m, 16);
    }
    const float riq = rsqrtf(sq / Dh + 1e-6f), rik = rsqrtf(sk / Dh + 1e-6f);
    float oq[8], ok[8];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float qa = x[2 * k] * riq * qg[2 * k], qb = x[2 * k + 1] * riq * qg[2 * k + 1];
      const float ka = y[2 * k] * rik * kg[2 * k], kb = y[2 * k + 1] * rik * kg[2 * k + 1];
      oq[2 * k] = qa * cs[k] - qb * sn[k];
      oq[2 * k + 1] = qa * sn[k] + qb * cs[k];
      ok[2 * k] = ka * cs[k] - kb * sn[k];
      ok[2 * k + 1] = ka * sn[k] + kb * cs[k];
    }
    if (hv) {
      const size_t o = ob + (size_t)h * N * Dh;
      st8f(Qh + o, oq);
      st8f(Kh + o, ok);
      *(uint4*)(Vh + o) = vv;
      if (lp == 0) {
        rq[(size_t)r * H + h] = riq;
        rk[(size_t)r * H + h] = rik;
      }
    }
  }
}

int qk_norm_rope_fwd(const void* proj, int ld, int act_dt, RowMap rm, Rope rp, Gains gn,
                     void* Qh, void* Kh, void* Vh, float* rinv_q, float* rinv_k, hipStream_t s) {
  if (rp.Dh > 128 || rp.Dh % 4) { set_error("qk_norm_rope: head_dim must be <= 128 and a multiple of 4"); return 1; }
  // RoPE pairs as one access each: even leading dimension, 8-byte aligned bases
  auto al8 = [](const void* p) { return ((uintptr_t)p & 7u) == 0; };
  if (act_dt == BF16 && rp.Dh == 128 && !(ld & 7) && al16(proj) && al16(Qh) && al16(Kh) && al16(Vh) &&
      al16(gn.q[0]) && al16(gn.q[1]) && al16(gn.k[0]) && al16(gn.k[1])) {
    hipLaunchKernelGGL(qk_norm_rope_fwd8_k, dim3((unsigned)((rm.rows() + 3) / 4)), dim3(256), 0, s,
                       (const uint16_t*)proj, ld, rm, rp, gn, (uint16_t*)Qh, (uint16_t*)Kh, (uint16_t*)Vh, rinv_q,
                       rinv_k);
    LAUNCH_OK("qk_norm_rope_fwd8");
    return 0;
  }
  if (!(ld & 1) && al8(proj) && al8(Qh) && al8(Kh) && al8(Vh)) {
    const dim3 grid((unsigned)((rm.rows() + 3) / 4));
    if (act_dt == BF16)
      hipLaunchKernelGGL(qk_norm_rope_fwd_row_k<uint16_t>, grid, dim3(256), 0, s, (const uint16_t*)proj, ld, rm, rp,
                         gn, (uint16_t*)Qh, (uint16_t*)Kh, (uint16_t*)Vh, rinv_q, rinv_k);
    else
      hipLaunchKernelGGL(qk_norm_rope_fwd_row_k<float>, grid, dim3(256), 0, s, (const float*)proj, ld, rm, rp, gn,
                         (float*)Qh, (float*)Kh, (float*)Vh, rinv_q, rinv_k);
    LAUNCH_OK("qk_norm_rope_fwd");
    return 0;
  }
  const int nitems = rm.rows() * rp.H;
  dim3 grid((nitems + 3) / 4);
  if (act_dt == BF16)
    hipLaunchKernelGGL(qk_norm_rope_fwd_k<uint16_t>, grid, dim3(256), 0, s, (const uint16_t*)proj, ld, rm, rp,
                       gn, (uint16_t*)Qh, (uint16_t*)Kh, (uint16_t*)Vh,
                       rinv_q, rinv_k, nitems);
  else
    hipLaunchKernelGGL(qk_norm_rope_fwd_k<float>, grid, dim3(256), 0, s, (const float*)proj, ld, rm, rp,
                       gn, (float*)Qh, (float*)Kh, (float*)Vh, rinv_q, rinv_k,
                       nitems);
  LAUNCH_OK("qk_norm_rope_fwd");
  return 0;
}

constexpr int QK_SUB = RED_ROWS / QK_PARTS;  // rows per block of the q/k norm backward

// two consecutive elements (an RoPE pair) as one 4- or 8-byte access
__device__ inline void ld2f(const uint16_t* p, float& a, float& c) {
  const uint32_t u = *(const uint32_t*)p;
  a = bf2f(u & 0xffffu);
  c = bf2f(u >> 16);
}
__device__ inline void ld2f(const float* p, float& a, float& c) {
  const float2 v = *(const float2*)p;
  a = v.x;
  c = v.y;
}
__device__ inline void st2f(uint16_t* p, float a, float c) {
  *(uint32_t*)p = (uint32_t)f2bf(a) | ((uint32_t)f2bf(c) << 16);
}
__device__ inline void st2f(float* p, float a, float c) { *(float2*)p = make_float2(a, c); }

// Forward, one wave per row: lane p owns RoPE pair p, whose rotation depends
// only on the token and is computed once per row; the heads are looped over
// with one pair access per operand.  Per head the arithmetic is that of
// qk_norm_rope_fwd_k (same lane sums, same products).
template <typename T>
__global__ __launch_bounds__(256) void qk_norm_rope_fwd_row_k(const T* __restrict__ proj, int ld, RowMap rm,
                                                              Rope rp, Gains gn, T* __restrict__ Qh,
                                                              T* __restrict__ Kh, T* __restrict__ Vh,
                                                              float* __restrict__ rq, float* __restrict__ rk) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rm.rows()) return;
  const int lane = threadIdx.x & 63;
  const int H = rp.H, Dh = rp.Dh, D = H * Dh, N = rm.nt + rm.ni;
  const bool act = lane < Dh / 2;
  const int p = act ? lane : 0;
  const T* pr = proj + (size_t)r * ld + 2 * p;
  const int st = r < rm.B * rm.nt ? 0 : 1;
  const T* qg = (const T*)gn.q[st];
  const T* kg = (const T*)gn.k[st];
  const float qga = act ? ldf(qg, 2 * p) : 0.f, qgb = act ? ldf(qg, 2 * p + 1) : 0.f;
  const float kga = act ? ldf(kg, 2 * p) : 0.f, kgb = act ? ldf(kg, 2 * p + 1) : 0.f;
  int b, j;
  tok_of_row(rm, r, b, j);
  float sn = 0.f, cs = 1.f;
  if (act) sincosf(rope_angle(rp, j, p), &sn, &cs);
  const size_t ob = ((size_t)b * H * N + j) * Dh + 2 * p;  // head h adds h * N * Dh
  for (int h = 0; h < H; ++h) {
    float q0 = 0.f, q1 = 0.f, k0 = 0.f, k1 = 0.f, v0 = 0.f, v1 = 0.f;
    if (act) {
      ld2f(pr + h * Dh, q0, q1);
      ld2f(pr + D + h * Dh, k0, k1);
      ld2f(pr + 2 * D + h * Dh, v0, v1);
    }
    const float riq = rsqrtf(wave_sum(q0 * q0 + q1 * q1) / Dh + 1e-6f);
    const float rik = rsqrtf(wave_sum(k0 * k0 + k1 * k1) / Dh + 1e-6f);
    if (lane == 0) {
      rq[(size_t)r * H + h] = riq;
      rk[(size_t)r * H + h] = rik;
    }
    if (act) {
      const float qa = q0 * riq * qga, qb = q1 * riq * qgb;
      const float ka = k0 * rik * kga, kb = k1 * rik * kgb;
      const size_t o = ob + (size_t)h * N * Dh;
      st2f(Qh + o, qa * cs - qb * sn, qa * sn + qb * cs);
      st2f(Kh + o, ka * cs - kb * sn, ka * sn + kb * cs);
      st2f(Vh + o, v0, v1);
    }
  }
}

// One wave per row (the rows of the sub-chunk dealt to the 4 waves), looping
// over the heads; lane p owns RoPE pair p, whose rotation depends only on the
// token and so is computed once per row.
template <typename T, typename TD>
__global__ __launch_bounds__(256) void qk_norm_rope_bwd_k(const TD* __restrict__ dQh, const TD* __restrict__ dKh,
                                                          const TD* __restrict__ dVh, const T* __restrict__ proj,
                                                          int ld, RowMap rm, Rope rp, Chunks ch, int c0,
                                                          Gains gn, const float* __restrict__ rq, const float* __restrict__ rk,
                                                          T* __restrict__ dproj, int ld_d, float* __restrict__ pgain) {
  __shared__ float red[4][4][64];
  // block = (chunk, sub-chunk of QK_SUB rows); gain partials per sub-chunk
  const int q = c0 + blockIdx.x;
  int r0, n, b;
  chunk_rows(ch, q, r0, n, b);
  const int st = r0 < ch.B * ch.nt ? 0 : 1;
  const int sub = (int)blockIdx.y;  // signed: an empty sub-chunk must get n <= 0
  r0 += sub * QK_SUB;
  n = min(QK_SUB, n - sub * QK_SUB);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int H = rp.H, Dh = rp.Dh, D = H * Dh, N = rm.nt + rm.ni;
  const bool act = lane < Dh / 2;
  const int p = act ? lane : 0;
  const T* qg = (const T*)gn.q[st];
  const T* kg = (const T*)gn.k[st];
  float gq0 = 0, gq1 = 0, gk0 = 0, gk1 = 0;
  const float qga = act ? ldf(qg, 2 * p) : 0.f, qgb = act ? ldf(qg, 2 * p + 1) : 0.f;
  const float kga = act ? ldf(kg, 2 * p) : 0.f, kgb = act ? ldf(kg, 2 * p + 1) : 0.f;
  const float inv_dh = 1.f / Dh;
  for (int rr = wave; rr < n; rr += 4) {
    const int r = r0 + rr;
    int bb, j;
    tok_of_row(rm, r, bb, j);
    float sn = 0.f, cs = 1.f;
    if (act) sincosf(rope_angle(rp, j, p), &sn, &cs);
    const T* pr = proj + (size_t)r * ld + 2 * p;
    T* dp = dproj + (size_t)r * ld_d + 2 * p;
    const size_t ob = ((size_t)bb * H * N + j) * Dh + 2 * p;  // head h adds h * N * Dh
    for (int h = 0; h < H; ++h) {
      const size_t o = ob + (size_t)h * N * Dh;
      float qa = 0, qc = 0, ka = 0, kc = 0, va = 0, vc = 0, x0 = 0, x1 = 0, y0 = 0, y1 = 0;
      if (act) {
        ld2f(dQh + o, qa, qc);
        ld2f(dKh + o, ka, kc);
        ld2f(dVh + o, va, vc);
        ld2f(pr + h * Dh, x0, x1);
        ld2f(pr + D + h * Dh, y0, y1);
      }
      const float riq = rq[(size_t)r * H + h], rik = rk[(size_t)r * H + h];
      // q: undo the rotation, then the RMS norm with gain
      const float d0 = qa * cs + qc * sn, d1 = -qa * sn + qc * cs;
      const float dotq = wave_sum(d0 * qga * x0 + d1 * qgb * x1);
      // k
      const float e0 = ka * cs + kc * sn, e1 = -ka * sn + kc * cs;
      const float dotk = wave_sum(e0 * kga * y0 + e1 * kgb * y1);
      if (act) {
        const float cq = riq * riq * riq * dotq * inv_dh, ck = rik * rik * rik * dotk * inv_dh;
        st2f(dp + h * Dh, d0 * qga * riq - x0 * cq, d1 * qgb * riq - x1 * cq);
        st2f(dp + D + h * Dh, e0 * kga * rik - y0 * ck, e1 * kgb * rik - y1 * ck);
        st2f(dp + 2 * D + h * Dh, va, vc);
        gq0 = fmaf(d0, x0 * riq, gq0);
        gq1 = fmaf(d1, x1 * riq, gq1);
        gk0 = fmaf(e0, y0 * rik, gk0);
        gk1 = fmaf(e1, y1 * rik, gk1);
      }
    }
  }
  red[wave][0][lane] = gq0;
  red[wave][1][lane] = gq1;
  red[wave][2][lane] = gk0;
  red[wave][3][lane] = gk1;
  __syncthreads();
  if (threadIdx.x < 64 && act) {
    float a[4] = {0, 0, 0, 0};
    for (int w = 0; w < 4; ++w)
      for (int k = 0; k < 4; ++k) a[k] += red[w][k][lane];
    float* out = pgain + ((size_t)q * QK_PARTS + sub) * 2 * rp.Dh;
    out[2 * p] = a[0];
    out[2 * p + 1] = a[1];
    out[rp.Dh + 2 * p] = a[2];
    out[rp.Dh + 2 * p + 1] = a[3];
  }
}

// The same backward for bf16 operands and head_dim 128 with 16-byte accesses:
// per step a wave takes four heads of its row, 16 lanes per head, each lane
// 4 RoPE pairs (8 consecutive elements).  The rotation of pair p is computed
// once per row by lane p and handed to the lanes that use it; the per-head
// sums run over the 16 lanes of the head.
__global__ __launch_bounds__(256) void qk_norm_rope_bwd8_k(const uint16_t* __restrict__ dQh,
                                                           const uint16_t* __restrict__ dKh,
                                                           const uint16_t* __restrict__ dVh,
                                                           const uint16_t* __restrict__ proj, int ld, RowMap rm,
                                                           Rope rp, Chunks ch, int c0, Gains gn,
                                                           const float* __restrict__ rq, const float* __restrict__ rk,
                                                           uint16_t* __restrict__ dproj, int ld_d,
                                                           float* __restrict__ pgain) {
  constexpr int Dh = 128;
  __shared__ float red[4][4][2 * Dh];  // [wave][head slot][q gains | k gains]
  const int q = c0 + blockIdx.x;
  int r0, n, b;
  chunk_rows(ch, q, r0, n, b);
  const int st = r0 < ch.B * ch.nt ? 0 : 1;
  const int sub = (int)blockIdx.y;  // signed: an empty sub-chunk must get n <= 0
  r0 += sub * QK_SUB;
  n = min(QK_SUB, n - sub * QK_SUB);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int hq = lane >> 4, lp = lane & 15, e0 = 8 * lp;
  const int H = rp.H, D = H * Dh, N = rm.nt + rm.ni;
  float qg[8], kg[8], gq[8], gk[8];
  ld8f((const uint16_t*)gn.q[st] + e0, qg);
  ld8f((const uint16_t*)gn.k[st] + e0, kg);
#pragma unroll
  for (int e = 0; e < 8; ++e) gq[e] = gk[e] = 0.f;
  constexpr float inv_dh = 1.f / Dh;
  for (int rr = wave; rr < n; rr += 4) {
    const int r = r0 + rr;
    int bb, j;
    tok_of_row(rm, r, bb, j);
    float sn0, cs0;
    sincosf(rope_angle(rp, j, lane), &sn0, &cs0);
    float cs[4], sn[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      cs[k] = __shfl(cs0, 4 * lp + k, 64);
      sn[k] = __shfl(sn0, 4 * lp + k, 64);
    }
    const uint16_t* pr = proj + (size_t)r * ld + e0;
    uint16_t* dp = dproj + (size_t)r * ld_d + e0;
    const size_t ob = ((size_t)bb * H * N + j) * Dh + e0;  // head h adds h * N * Dh
    for (int h0 = 0; h0 < H; h0 += 4) {
      const int h = h0 + hq;
      const bool hv = h < H;
      const int hh = hv ? h : 0;  // lanes past the last head compute on head 0, store nothing
      const size_t o = ob + (size_t)hh * N * Dh;
      float qa[8], ka[8], x[8], y[8];
      ld8f(dQh + o, qa);
      ld8f(dKh + o, ka);
      ld8f(pr + hh * Dh, x);
      ld8f(pr + D + hh * Dh, y);
      const uint4 vv = *(const uint4*)(dVh + o);
      const float riq = rq[(size_t)r * H + hh], rik = rk[(size_t)r * H + hh];
      // undo the rotation
      float dq[8], dk[8];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        dq[2 * k] = qa[2 * k] * cs[k] + qa[2 * k + 1] * sn[k];
        dq[2 * k + 1] = -qa[2 * k] * sn[k] + qa[2 * k + 1] * cs[k];
        dk[2 * k] = ka[2 * k] * cs[k] + ka[2 * k + 1] * sn[k];
        dk[2 * k + 1] = -ka[2 * k] * sn[k] + ka[2 * k + 1] * cs[k];
      }
      float sq = 0.f, sk = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        sq = fmaf(dq[e] * qg[e], x[e], sq);
        sk = fmaf(dk[e] * kg[e], y[e], sk);
      }
#pragma unroll
      for (int m = 8; m > 0; m >>= 1) {
        sq += __shfl_xor(sq, m, 16);
        sk += __shfl_xor(sk, m, 16);
      }
      const float cq = riq * riq * riq * sq * inv_dh, ck = rik * rik * rik * sk * inv_dh;
      float oq[8], ok[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        oq[e] = dq[e] * qg[e] * riq - x[e] * cq;
        ok[e] = dk[e] * kg[e] * rik - y[e] * ck;
      }
      if (hv) {
        st8f(dp + h * Dh, oq);
        st8f(dp + D + h * Dh, ok);
        *(uint4*)(dp + 2 * D + h * Dh) = vv;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          gq[e] = fmaf(dq[e], x[e] * riq, gq[e]);
          gk[e] = fmaf(dk[e], y[e] * rik, gk[e]);
        }
      }
    }
  }
  // gain partials: the 16 head slots of the block (4 waves x 4) added in order
  float* const rw = &red[wave][hq][0];
  *(float4*)(rw + e0) = make_float4(gq[0], gq[1], gq[2], gq[3]);
  *(float4*)(rw + e0 + 4) = make_float4(gq[4], gq[5], gq[6], gq[7]);
  *(float4*)(rw + Dh + e0) = make_float4(gk[0], gk[1], gk[2], gk[3]);
  *(float4*)(rw + Dh + e0 + 4) = make_float4(gk[4], gk[5], gk[6], gk[7]);
  __syncthreads();
  const int c = threadIdx.x;  // 256 threads = 2 Dh gain columns
  float a = 0.f;
#pragma unroll
  for (int w = 0; w < 4; ++w)
#pragma unroll
    for (int k = 0; k < 4; ++k) a += red[w][k][c];
  pgain[((size_t)q * QK_PARTS + sub) * 2 * Dh + c] = a;
}

int qk_norm_rope_bwd(const void* dQh, const void* dKh, const void* dVh, int dt_d, const void* proj, int ld,
                     int act_dt, RowMap rm, Rope rp, Gains gn, const float* rinv_q,
                     const float* rinv_k, void* dproj, int ld_d, float* part_gain, hipStream_t s) {
  if (rp.Dh > 128 || rp.Dh % 4) { set_error("qk_norm_rope_bwd: head_dim"); return 1; }
  // RoPE pairs are read and written as one access: even leading dimensions,
  // 8-byte aligned bases
  auto al8 = [](const void* p) { return ((uintptr_t)p & 7u) == 0; };
  if ((ld | ld_d) & 1 || !al8(dQh) || !al8(dKh) || !al8(dVh) || !al8(proj) || !al8(dproj)) {
    set_error("qk_norm_rope_bwd: operands must be 8-byte aligned with even leading dimensions");
    return 1;
  }
  int c0, nc;
  if (chunk_range(rm, 0, rm.rows(), &c0, &nc)) return 1;
  Chunks ch{rm.B, rm.nt, rm.ni, RED_ROWS};
  if (act_dt == BF16 && dt_d == BF16 && rp.Dh == 128 && !((ld | ld_d) & 7) && al16(dQh) && al16(dKh) && al16(dVh) &&
      al16(proj) && al16(dproj) && al16(gn.q[0]) && al16(gn.q[1]) && al16(gn.k[0]) && al16(gn.k[1])) {
    hipLaunchKernelGGL(qk_norm_rope_bwd8_k, dim3(nc, QK_PARTS), dim3(256), 0, s, (const uint16_t*)dQh,
                       (const uint16_t*)dKh, (const uint16_t*)dVh, (const uint16_t*)proj, ld, rm, rp, ch, c0, gn,
                       rinv_q, rinv_k, (uint16_t*)dproj, ld_d, part_gain);
    LAUNCH_OK("qk_norm_rope_bwd8");
    return 0;
  }
#define QKB(T, TD)                                                                                            \
  hipLaunchKernelGGL((qk_norm_rope_bwd_k<T, TD>), dim3(nc, QK_PARTS), dim3(256), 0, s, (const TD*)dQh, (const TD*)dKh,     \
                     (const TD*)dVh, (const T*)proj, ld, rm, rp, ch, c0, gn, rinv_q, rinv_k, \
                     (T*)dproj, ld_d, part_gain)
  if (act_dt == BF16 && dt_d == BF16) QKB(uint16_t, uint16_t);
  else if (act_dt == BF16) QKB(uint16_t, float);
  else if (dt_d == BF16) QKB(float, uint16_t);
  else QKB(float, float);
#undef QKB
  LAUNCH_OK("qk_norm_rope_bwd");
  return 0;
}

// ================================================================ reductions
template <typename T>
__global__ __launch_bounds__(256) void colsum_k(const T* __restrict__ X, int ld, int N, Chunks ch, int c0,
                                                float* __restrict__ part) {
  const int q = c0 + blockIdx.x;
  int r0, n, b;
  chunk_rows(ch, q, r0, n, b);
  for (int c = threadIdx.x; c < N; c += 256) {
    float s = 0.f;
    for (int rr = 0; rr < n; ++rr) s += ldf(X, (size_t)(r0 + rr) * ld + c);
    part[(size_t)q * N + c] = s;
  }
}

// 8 consecutive columns per thread, 16-byte loads down the chunk's rows
template <typename T>
__global__ __launch_bounds__(256) void colsum_vec_k(const T* __restrict__ X, int ld, int N, Chunks ch, int c0,
                                                    float* __restrict__ part) {
  const int q = c0 + blockIdx.x;
  int r0, n, b;
  chunk_rows(ch, q, r0, n, b);
  const int c = (blockIdx.y * 256 + threadIdx.x) * 8;
  if (c >= N) return;
  float sacc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll 4
  for (int rr = 0; rr < n; ++rr) {
    float v[8];
    ld8f(X + (size_t)(r0 + rr) * ld + c, v);
#pragma unroll
    for (int e = 0; e < 8; ++e) sacc[e] += v[e];
  }
  st8f(part + (size_t)q * N + c, sacc);
}

int colsum_partials(const void* X, int dt, int ld, int N, RowMap rm, int row0, int nrows, float* part,
                    hipStream_t s) {
  int c0, nc;
  if (chunk_range(rm, row0, nrows, &c0, &nc)) return 1;
  if (nc == 0) return 0;
  Chunks ch{rm.B, rm.nt, rm.ni, RED_ROWS};
  if (N % 8 == 0 && ld % 8 == 0 && al16(X) && al16(part)) {
    dim3 grid(nc, (N + 2047) / 2048);
    if (dt == BF16)
      hipLaunchKernelGGL(colsum_vec_k<uint16_t>, grid, dim3(256), 0, s, (const uint16_t*)X, ld, N, ch, c0, part);
    else
      hipLaunchKernelGGL(colsum_vec_k<float>, grid, dim3(256), 0, s, (const float*)X, ld, N, ch, c0, part);
    LAUNCH_OK("colsum_vec");
    return 0;
  }
  if (dt == BF16)
    hipLaunchKernelGGL(colsum_k<uint16_t>, dim3(nc), dim3(256), 0, s, (const uint16_t*)X, ld, N, ch, c0, part);
  else
    hipLaunchKernelGGL(colsum_k<float>, dim3(nc), dim3(256), 0, s, (const float*)X, ld, N, ch, c0, part);
  LAUNCH_OK("colsum");
  return 0;
}

// Per sample: the sample's chunks inside [c0, c0 + nc) form at most two runs
// (its text chunks, its image chunks); 32 columns x 8 slices per block.
// Column sums of chunk partials are latency-bound (few columns, many chunks):
// a block takes 64 consecutive columns (one 256-byte row segment per wave
// load) and 16 chunk slices (slice k sums chunks k, k+16, ...; loads unrolled
// so several are in flight), and adds the 16 slice sums in slice order
// (deterministic).
constexpr int RC_COLS = 64, RC_SL = 16;

__device__ inline float slice_total(float acc, float (*sh)[RC_COLS + 1]) {
  const int cl = threadIdx.x % RC_COLS, sl = threadIdx.x / RC_COLS;
  sh[sl][cl] = acc;
  __syncthreads();
  float t = 0.f;
  if (sl == 0) {
#pragma unroll
    for (int k = 0; k < RC_SL; ++k) t += sh[k][cl];
  }
  return t;
}

__global__ __launch_bounds__(1024) void reduce_per_sample_k(const float* __restrict__ part, int N, Chunks ch, int c0,
                                                            int nc, float* __restrict__ out, int out_stride,
                                                            int out_off) {
  __shared__ float sh[RC_SL][RC_COLS + 1];
  const int b = blockIdx.y;
  const int cl = threadIdx.x % RC_COLS, sl = threadIdx.x / RC_COLS;
  const int c = blockIdx.x * RC_COLS + cl;
  const int ct = ch.ct(), ci = ch.ci();
  const int runs[2][2] = {{b * ct, b * ct + ct}, {ch.B * ct + b * ci, ch.B * ct + b * ci + ci}};
  float acc = 0.f;
  if (c < N)
    for (int r = 0; r < 2; ++r) {
      const int lo = max(runs[r][0], c0), hi = min(runs[r][1], c0 + nc);
#pragma unroll 4
      for (int q = lo + sl; q < hi; q += RC_SL) acc += part[(size_t)q * N + c];
    }
  const float t = slice_total(acc, sh);
  if (sl == 0 && c < N) out[(size_t)b * out_stride + out_off + c] = t;
}

int reduce_per_sample(const float* part, int N, RowMap rm, int row0, int nrows, float* out, int out_stride,
                      int out_off, hipStream_t s, int R) {
  int c0, nc;
  if (chunk_range(rm, row0, nrows, &c0, &nc, R)) return 1;
  Chunks ch{rm.B, rm.nt, rm.ni, R};
  hipLaunchKernelGGL(reduce_per_sample_k, dim3((N + RC_COLS - 1) / RC_COLS, rm.B), dim3(RC_COLS * RC_SL), 0, s, part,
                     N, ch, c0, nc, out, out_stride, out_off);
  LAUNCH_OK("reduce_per_sample");
  return 0;
}

// g[c] (+)= sum over chunks [chunk0, chunk0 + nchunk) of part[q * ld + c];
// beta * g is added once, after the slices.
template <typename TG>
__global__ __launch_bounds__(1024) void reduce_to_grad_k(const float* __restrict__ part, int ld, int chunk0,
                                                         int nchunk, int N, TG* __restrict__ g, float beta) {
  __shared__ float sh[RC_SL][RC_COLS + 1];
  const int cl = threadIdx.x % RC_COLS, sl = threadIdx.x / RC_COLS;
  const int c = blockIdx.x * RC_COLS + cl;
  float acc = 0.f;
  if (c < N) {
#pragma unroll 4
    for (int q = chunk0 + sl; q < chunk0 + nchunk; q += RC_SL) acc += part[(size_t)q * ld + c];
  }
  float t = slice_total(acc, sh);
  if (sl == 0 && c < N) {
    if (beta != 0.f) t += beta * ldf(g, c);
    stf(g, c, t);
  }
}

int reduce_to_grad(const float* part, int ld, int chunk0, int nchunk, int N, void* g, int g_dt,
                   float beta, hipStream_t s) {
  dim3 grid((N + RC_COLS - 1) / RC_COLS);
  if (g_dt == BF16)
    hipLaunchKernelGGL(reduce_to_grad_k<uint16_t>, grid, dim3(RC_COLS * RC_SL), 0, s, part, ld, chunk0, nchunk, N,
                       (uint16_t*)g, beta);
  else
    hipLaunchKernelGGL(reduce_to_grad_k<float>, grid, dim3(RC_COLS * RC_SL), 0, s, part, ld, chunk0, nchunk, N,
                       (float*)g, beta);
  LAUNCH_OK("reduce_to_grad");
  return 0;
}

// ---- reduction jobs in one launch ----
struct RedJobs {
  RedJob j[RED_MAX_JOBS];
  int n;
};

RedJob per_sample_job(const float* part, int N, RowMap rm, int row0, int nrows, float* out, int out_stride,
                      int out_off, int R) {
  RedJob r;
  r.part = part;
  r.ld = r.N = N;
  r.kind = 0;
  r.ch = Chunks{rm.B, rm.nt, rm.ni, R};
  if (chunk_range(rm, row0, nrows, &r.c0, &r.nc, R)) r.N = -1;  // rejected by reduce_jobs
  r.out = out;
  r.out_stride = out_stride;
  r.out_off = out_off;
  return r;
}

RedJob to_grad_job(const float* part, int ld, int chunk0, int nchunk, int N, void* g, int g_dt, float beta) {
  RedJob r;
  r.part = part;
  r.ld = ld;
  r.N = N;
  r.kind = 1;
  r.c0 = chunk0;
  r.nc = nchunk;
  r.g = g;
  r.g_dt = g_dt;
  r.beta = beta;
  return r;
}

// Block x of the launch belongs to the job whose block range holds it; inside
// the job, the block's column group and (per sample) its sample follow the
// grids of reduce_per_sample_k and reduce_to_grad_k, and so do the sums.
__global__ __launch_bounds__(1024) void reduce_jobs_k(RedJobs js) {
  __shared__ float sh[RC_SL][RC_COLS + 1];
  int k = 0;
  while (k + 1 < js.n && (int)blockIdx.x >= js.j[k + 1].blk0) ++k;
  const RedJob& J = js.j[k];
  const int cl = threadIdx.x % RC_COLS, sl = threadIdx.x / RC_COLS;
  const int ncol = (J.N + RC_COLS - 1) / RC_COLS;
  const int local = (int)blockIdx.x - J.blk0;
  const int c = (local % ncol) * RC_COLS + cl;
  float acc = 0.f;
  if (J.kind == 0) {
    const int b = local / ncol;
    const int ct = J.ch.ct(), ci = J.ch.ci();
    const int runs[2][2] = {{b * ct, b * ct + ct}, {J.ch.B * ct + b * ci, J.ch.B * ct + b * ci + ci}};
    if (c < J.N)
      for (int r = 0; r < 2; ++r) {
        const int lo = max(runs[r][0], J.c0), hi = min(runs[r][1], J.c0 + J.nc);
#pragma unroll 4
        for (int q = lo + sl; q < hi; q += RC_SL) acc += J.part[(size_t)q * J.ld + c];
      }
    const float t = slice_total(acc, sh);
    if (sl == 0 && c < J.N) J.out[(size_t)b * J.out_stride + J.out_off + c] = t;
  } else {
    if (c < J.N) {
#pragma unroll 4
      for (int q = J.c0 + sl; q < J.c0 + J.nc; q += RC_SL) acc += J.part[(size_t)q * J.ld + c];
    }
    float t = slice_total(acc, sh);
    if (sl == 0 && c < J.N) {
      if (J.g_dt == BF16) {
        if (J.beta != 0.f) t += J.beta * ldf((const uint16_t*)J.g, c);
        stf((uint16_t*)J.g, c, t);
      } else {
        if (J.beta != 0.f) t += J.beta * ldf((const float*)J.g, c);
        stf((float*)J.g, c, t);
      }
    }
  }
}

int reduce_jobs(const RedJob* jobs, int n, hipStream_t s) {
  if (n < 1 || n > RED_MAX_JOBS) { set_error("reduce_jobs: 1..8 jobs"); return 1; }
  RedJobs js;
  js.n = n;
  int blk = 0;
  for (int k = 0; k < n; ++k) {
    js.j[k] = jobs[k];
    const RedJob& J = js.j[k];
    if (J.N <= 0 || !J.part || (J.kind == 0 && (!J.out || J.ld != J.N)) || (J.kind == 1 && !J.g) || J.kind < 0 ||
        J.kind > 1) {
      set_error("reduce_jobs: invalid job");
      return 1;
    }
    js.j[k].blk0 = blk;
    blk += (J.N + RC_COLS - 1) / RC_COLS * (J.kind == 0 ? J.ch.B : 1);
  }
  hipLaunchKernelGGL(reduce_jobs_k, dim3(blk), dim3(RC_COLS * RC_SL), 0, s, js);
  LAUNCH_OK("reduce_jobs");
  return 0;
}

// ================================================================ misc
template <typename T>
__global__ void patchify_k(const T* __restrict__ z, int B, int C, int Hh, int Ww, int p, T* __restrict__ out,
                           bool inverse) {
  const size_t n = (size_t)B * C * Hh * Ww;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int gw = Ww / p, gh = Hh / p, pd = C * p * p;
  // i indexes the token-major tensor [B][gh*gw][pd]
  const int f = (int)(i % pd);
  const size_t tok = i / pd;
  const int b = (int)(tok / ((size_t)gh * gw));
  const int t = (int)(tok % ((size_t)gh * gw));
  const int r = t / gw, c = t % gw;
  const int ch = f / (p * p), py = (f / p) % p, px = f % p;
  const size_t zi = (((size_t)b * C + ch) * Hh + r * p + py) * Ww + c * p + px;
  if (!inverse) out[i] = z[zi];
  else out[zi] = z[i];
}

int patchify(const void* z, int dt, int B, int C, int Hh, int Ww, int p, void* out, hipStream_t s) {
  const size_t n = (size_t)B * C * Hh * Ww;
  dim3 grid((unsigned)((n + 255) / 256));
  if (dt == BF16)
    hipLaunchKernelGGL(patchify_k<uint16_t>, grid, dim3(256), 0, s, (const uint16_t*)z, B, C, Hh, Ww, p,
                       (uint16_t*)out, false);
  else
    hipLaunchKernelGGL(patchify_k<float>, grid, dim3(256), 0, s, (const float*)z, B, C, Hh, Ww, p, (float*)out,
                       false);
  LAUNCH_OK("patchify");
  return 0;
}

int unpatchify(const void* x, int dt, int B, int C, int Hh, int Ww, int p, void* z, hipStream_t s) {
  const size_t n = (size_t)B * C * Hh * Ww;
  dim3 grid((unsigned)((n + 255) / 256));
  if (dt == BF16)
    hipLaunchKernelGGL(patchify_k<uint16_t>, grid, dim3(256), 0, s, (const uint16_t*)x, B, C, Hh, Ww, p,
                       (uint16_t*)z, true);
  else
    hipLaunchKernelGGL(patchify_k<float>, grid, dim3(256), 0, s, (const float*)x, B, C, Hh, Ww, p, (float*)z, true);
  LAUNCH_OK("unpatchify");
  return 0;
}

__global__ void convert_k(const void* x, int dti, void* y, int dto, size_t n) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) st_any(y, dto, i, ld_any(x, dti, i));
}
// 8 elements per thread: 16- and 32-byte accesses (the same conversions as
// convert_k, so the same bits)
template <typename TI, typename TO>
__global__ void convert8_k(const TI* __restrict__ x, TO* __restrict__ y, size_t n8) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n8) {
    float v[8];
    ld8f(x + 8 * i, v);
    st8f(y + 8 * i, v);
  }
}
int convert(const void* x, int dt_in, void* y, int dt_out, size_t n, hipStream_t s) {
  if (!n) return 0;
  size_t done = 0;
  if (al16(x) && al16(y) && n >= 8) {
    const size_t n8 = n / 8;
    const dim3 grid((unsigned)((n8 + 255) / 256));
    if (dt_in == BF16 && dt_out == F32)
      hipLaunchKernelGGL((convert8_k<uint16_t, float>), grid, dim3(256), 0, s, (const uint16_t*)x, (float*)y, n8);
    else if (dt_in == F32 && dt_out == BF16)
      hipLaunchKernelGGL((convert8_k<float, uint16_t>), grid, dim3(256), 0, s, (const float*)x, (uint16_t*)y, n8);
    else if (dt_in == BF16)
      hipLaunchKernelGGL((convert8_k<uint16_t, uint16_t>), grid, dim3(256), 0, s, (const uint16_t*)x, (uint16_t*)y, n8);
    else
      hipLaunchKernelGGL((convert8_k<float, float>), grid, dim3(256), 0, s, (const float*)x, (float*)y, n8);
    LAUNCH_OK("convert");
    done = n8 * 8;
  }
  if (done < n) {
    const size_t r = n - done;
    hipLaunchKernelGGL(convert_k, dim3((unsigned)((r + 255) / 256)), dim3(256), 0, s,
                       (const void*)((const char*)x + done * dsize(dt_in)), dt_in,
                       (void*)((char*)y + done * dsize(dt_out)), dt_out, r);
    LAUNCH_OK("convert");
  }
  return 0;
}

__global__ void fill_zero_k(uint32_t* p, size_t n) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}
int fill_zero(void* x, size_t bytes, hipStream_t s) {
  if (bytes % 4) { set_error("fill_zero: size must be a multiple of 4 bytes"); return 1; }
  const size_t n = bytes / 4;
  if (!n) return 0;
  hipLaunchKernelGGL(fill_zero_k, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, (uint32_t*)x, n);
  LAUNCH_OK("fill_zero");
  return 0;
}

// ================================================================ aggregation
// Each thread owns 8 consecutive elements per grid-stride step: W 16-byte (bf16)
// or 32-byte (fp32) loads, fp32 FMA accumulation in j order, one rounding on
// store.  HBM traffic per element: W reads + 2 writes.
template <typename TI, typename TO>
__global__ __launch_bounds__(256) void aggregate_k(AggArgs a) {
  const size_t nv = a.n / 8;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t v = (size_t)blockIdx.x * blockDim.x + threadIdx.x; v < nv; v += stride) {
    float sb[8], sc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) sb[e] = sc[e] = 0.f;
    for (int j = 0; j < a.W; ++j) {
      float x[8];
      const TI* p = (const TI*)a.s[j] + v * 8;
      if constexpr (sizeof(TI) == 2) {
        const uint4 u = *(const uint4*)p;
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) { x[2 * e] = bf2f(w[e] & 0xffff); x[2 * e + 1] = bf2f(w[e] >> 16); }
      } else {
        const float4 u0 = *(const float4*)p, u1 = *(const float4*)(p + 4);
        x[0] = u0.x; x[1] = u0.y; x[2] = u0.z; x[3] = u0.w;
        x[4] = u1.x; x[5] = u1.y; x[6] = u1.z; x[7] = u1.w;
      }
      const float wb = a.wb[j], wc = a.wc[j];
#pragma unroll
      for (int e = 0; e < 8; ++e) { sb[e] = fmaf(wb, x[e], sb[e]); sc[e] = fmaf(wc, x[e], sc[e]); }
    }
    const size_t e0 = v * 8;
    // the destinations of this element's segment; a null destination skips
    // that composite (one endpoint of the sequential variant)
    const bool lo = e0 < a.split;
    TO* const db0 = (TO*)(lo ? a.base0 : a.base1);
    TO* const dc0 = (TO*)(lo ? a.corr0 : a.corr1);
    const size_t off = lo ? e0 : e0 - a.split;
    TO* const db = db0 ? db0 + off : nullptr;
    TO* const dc = dc0 ? dc0 + off : nullptr;
    if constexpr (sizeof(TO) == 2) {
      uint4 ub, uc;
      ub.x = f2bf(sb[0]) | ((uint32_t)f2bf(sb[1]) << 16); ub.y = f2bf(sb[2]) | ((uint32_t)f2bf(sb[3]) << 16);
      ub.z = f2bf(sb[4]) | ((uint32_t)f2bf(sb[5]) << 16); ub.w = f2bf(sb[6]) | ((uint32_t)f2bf(sb[7]) << 16);
      uc.x = f2bf(sc[0]) | ((uint32_t)f2bf(sc[1]) << 16); uc.y = f2bf(sc[2]) | ((uint32_t)f2bf(sc[3]) << 16);
      uc.z = f2bf(sc[4]) | ((uint32_t)f2bf(sc[5]) << 16); uc.w = f2bf(sc[6]) | ((uint32_t)f2bf(sc[7]) << 16);
      if (db) *(uint4*)db = ub;
      if (dc) *(uint4*)dc = uc;
    } else {
      if (db) {
        *(float4*)db = make_float4(sb[0], sb[1], sb[2], sb[3]);
        *(float4*)(db + 4) = make_float4(sb[4], sb[5], sb[6], sb[7]);
      }
      if (dc) {
        *(float4*)dc = make_float4(sc[0], sc[1], sc[2], sc[3]);
        *(float4*)(dc + 4) = make_float4(sc[4], sc[5], sc[6], sc[7]);
      }
    }
  }
}

// scalar tail / unaligned path
__global__ void aggregate_scalar_k(AggArgs a, size_t e_begin) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t e = e_begin + (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < a.n; e += stride) {
    float sb = 0.f, sc = 0.f;
    for (int j = 0; j < a.W; ++j) {
      const float x = ld_any(a.s[j], a.in_dt, e);
      sb = fmaf(a.wb[j], x, sb);
      sc = fmaf(a.wc[j], x, sc);
    }
    if (e < a.split) {
      if (a.base0) st_any(a.base0, a.out_dt, e, sb);
      if (a.corr0) st_any(a.corr0, a.out_dt, e, sc);
    } else {
      if (a.base1) st_any(a.base1, a.out_dt, e - a.split, sb);
      if (a.corr1) st_any(a.corr1, a.out_dt, e - a.split, sc);
    }
  }
}

int aggregate(const AggArgs& a, hipStream_t s) {
  if (a.W < 1 || a.W > 64) { set_error("aggregate: W must be 1..64"); return 1; }
  if (a.n == 0) return 0;
  bool vec = (a.n % 8 == 0) && (a.split % 8 == 0);
  const uintptr_t al = (uintptr_t)a.base0 | (uintptr_t)a.base1 | (uintptr_t)a.corr0 | (uintptr_t)a.corr1;
  vec = vec && (al % 16 == 0);
  for (int j = 0; j < a.W; ++j) vec = vec && ((uintptr_t)a.s[j] % 16 == 0);
  const int pi = prof_begin(PROF_AGGREGATE);
  if (vec) {
    const size_t nv = a.n / 8;
    const unsigned grid = (unsigned)std::min<size_t>((nv + 255) / 256, 256 * 16);
#define AGG(TI, TO) launch(aggregate_k<TI, TO>, dim3(grid), dim3(256), 0u, s, a)
    if (a.in_dt == BF16 && a.out_dt == BF16) AGG(uint16_t, uint16_t);
    else if (a.in_dt == BF16) AGG(uint16_t, float);
    else if (a.out_dt == BF16) AGG(float, uint16_t);
    else AGG(float, float);
#undef AGG
  } else {
    const unsigned grid = (unsigned)std::min<size_t>((a.n + 255) / 256, 256 * 16);
    launch(aggregate_scalar_k, dim3(grid), dim3(256), 0u, s, a, (size_t)0);
  }
  prof_end(pi, (double)a.n * ((double)a.W * dsize(a.in_dt) + 2.0 * dsize(a.out_dt)));
  LAUNCH_OK("aggregate");
  return 0;
}

// ================================================================ group scores
// Pair products (i <= j) accumulated in fp64; one partial row per block, then a
// single block sums partials in block order (deterministic).
constexpr int SC_BLOCKS = 512;
size_t score_part_doubles(int W) { return (size_t)SC_BLOCKS * (W * (W + 1) / 2); }

template <int W>
__global__ __launch_bounds__(256) void scores_pass1_k(ScoreArgs a, double* part) {
  constexpr int P = W * (W + 1) / 2;
  __shared__ double sh[4][P];
  double acc[P];
#pragma unroll
  for (int k = 0; k < P; ++k) acc[k] = 0.0;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < a.n; e += stride) {
    double x[W];
#pragma unroll
    for (int i = 0; i < W; ++i) x[i] = (double)ld_any(a.h[i], a.dt, e);
    int k = 0;
#pragma unroll
    for (int i = 0; i < W; ++i)
#pragma unroll
      for (int j = i; j < W; ++j) acc[k++] += x[i] * x[j];
  }
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
#pragma unroll
  for (int k = 0; k < P; ++k) {
    double v = acc[k];
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    if (lane == 0) sh[wv][k] = v;
  }
  __syncthreads();
  for (int k = threadIdx.x; k < P; k += 256)
    part[(size_t)blockIdx.x * P + k] = sh[0][k] + sh[1][k] + sh[2][k] + sh[3][k];
}

__global__ void scores_pass2_k(const double* part, int nblk, int W, double* score) {
  __shared__ double tot[64];
  const int P = W * (W + 1) / 2;
  for (int k = threadIdx.x; k < P; k += blockDim.x) {
    double s = 0.0;
    for (int b = 0; b < nblk; ++b) s += part[(size_t)b * P + k];
    tot[k] = s;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    // index of (i, j), i <= j, in the row-major upper triangle
    auto idx = [W](int i, int j) { return i * W - i * (i - 1) / 2 + (j - i); };
    double s = 0.0;
    int cnt = 0;
    for (int i = 0; i < W; ++i)
      for (int j = i + 1; j < W; ++j) {
        s += tot[idx(i, j)] / (sqrt(tot[idx(i, i)]) * sqrt(tot[idx(j, j)]));
        ++cnt;
      }
    *score = s / cnt;
  }
}

int group_scores(const ScoreArgs& a, double* part, double* score_dev, hipStream_t s) {
  if (a.W < 2 || a.W > 8) { set_error("group_scores: W must be 2..8"); return 1; }
  if (a.n == 0) { set_error("group_scores: empty vectors"); return 1; }
  const unsigned grid = SC_BLOCKS;
  switch (a.W) {
#define SCW(w) case w: hipLaunchKernelGGL(scores_pass1_k<w>, dim3(grid), dim3(256), 0, s, a, part); break;
    SCW(2) SCW(3) SCW(4) SCW(5) SCW(6) SCW(7) SCW(8)
#undef SCW
  }
  LAUNCH_OK("group_scores_pass1");
  hipLaunchKernelGGL(scores_pass2_k, dim3(1), dim3(64), 0, s, part, (int)grid, a.W, score_dev);
  LAUNCH_OK("group_scores_pass2");
  return 0;
}


// ============================================================ gradient compare
// Gradient-quality sums for cos(a, b) and |a| / |b|: a.b, a.a, b.b over n
// elements, fp64 accumulation.  Pass 1: every thread walks 8-element vectors
// (16- or 32-byte loads) grid-stride, a block writes its three partials; pass
// 2: one block adds the block partials in block order (deterministic).
// HBM traffic: one read of each vector.
size_t compare_part_doubles() { return (size_t)CMP_BLOCKS * 3; }

template <typename T>
__device__ __forceinline__ void load8f(const T* p, float* x) {
  if constexpr (sizeof(T) == 2) {
    const uint4 u = *(const uint4*)p;
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) { x[2 * e] = bf2f(w[e] & 0xffff); x[2 * e + 1] = bf2f(w[e] >> 16); }
  } else {
    const float4 u0 = *(const float4*)p, u1 = *(const float4*)(p + 4);
    x[0] = u0.x; x[1] = u0.y; x[2] = u0.z; x[3] = u0.w;
    x[4] = u1.x; x[5] = u1.y; x[6] = u1.z; x[7] = u1.w;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void compare_pass1_k(const T* a, const T* b, size_t n, double* part) {
  __shared__ double sh[4][3];
  double ab = 0.0, aa = 0.0, bb = 0.0;
  const size_t nv = n / 8, stride = (size_t)gridDim.x * blockDim.x;
  const size_t t0 = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (size_t v = t0; v < nv; v += stride) {
    float x[8], y[8];
    load8f<T>(a + v * 8, x);
    load8f<T>(b + v * 8, y);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      ab = fma((double)x[e], (double)y[e], ab);
      aa = fma((double)x[e], (double)x[e], aa);
      bb = fma((double)y[e], (double)y[e], bb);
    }
  }
  // ragged tail (n % 8 elements), thread 0 of block 0
  if (t0 == 0)
    for (size_t e = nv * 8; e < n; ++e) {
      const double x = ldf(a, e), y = ldf(b, e);
      ab = fma(x, y, ab); aa = fma(x, x, aa); bb = fma(y, y, bb);
    }
  double v3[3] = {ab, aa, bb};
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    double v = v3[k];
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    if (lane == 0) sh[wv][k] = v;
  }
  __syncthreads();
  if (threadIdx.x < 3) part[(size_t)blockIdx.x * 3 + threadIdx.x] = sh[0][threadIdx.x] + sh[1][threadIdx.x] +
                                                                     sh[2][threadIdx.x] + sh[3][threadIdx.x];
}

__global__ void compare_pass2_k(const double* part, int nblk, double* out) {
  if (threadIdx.x < 3) {
    double s = 0.0;
    for (int b = 0; b < nblk; ++b) s += part[(size_t)b * 3 + threadIdx.x];
    out[threadIdx.x] = s;
  }
}

int grad_compare(const void* a, const void* b, size_t n, int dt, double* part, double* out_dev, hipStream_t s) {
  if (!a || !b || n == 0) { set_error("grad_compare: empty or null vectors"); return 1; }
  if ((((uintptr_t)a | (uintptr_t)b) & 15) != 0) { set_error("grad_compare: vectors must be 16-byte aligned"); return 1; }
  const size_t nv = n / 8;
  const unsigned grid = (unsigned)std::max<size_t>(1, std::min<size_t>((nv + 255) / 256, CMP_BLOCKS));
  const int pi = prof_begin(PROF_COMPARE);
  if (dt == BF16) launch(compare_pass1_k<uint16_t>, dim3(grid), dim3(256), 0u, s, (const uint16_t*)a, (const uint16_t*)b, n,
                         part);
  else launch(compare_pass1_k<float>, dim3(grid), dim3(256), 0u, s, (const float*)a, (const float*)b, n, part);
  prof_end(pi, 2.0 * (double)n * dsize(dt));
  LAUNCH_OK("grad_compare_pass1");
  hipLaunchKernelGGL(compare_pass2_k, dim3(1), dim3(64), 0, s, part, (int)grid, out_dev);
  LAUNCH_OK("grad_compare_pass2");
  return 0;
}


// ---- non-finite scan: elements whose exponent bits are all ones (NaN, +-Inf),
// counted exactly in 64-bit integers: per-block counts, then one sum.
template <typename T>
__device__ __forceinline__ unsigned nonfinite8(const T* p) {
  const uint4 u = *(const uint4*)p;
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
  unsigned c = 0;
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int e = 0; e < 4; ++e) c += ((w[e] & 0x7f80u) == 0x7f80u) + ((w[e] & 0x7f800000u) == 0x7f800000u);
  } else {
    const uint4 v = *(const uint4*)(p + 4);
    const uint32_t z[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) c += ((w[e] & 0x7f800000u) == 0x7f800000u) + ((z[e] & 0x7f800000u) == 0x7f800000u);
  }
  return c;
}

template <typename T>
__global__ __launch_bounds__(256) void nonfinite_pass1_k(const T* x, size_t n, unsigned long long* part) {
  __shared__ unsigned long long sh[4];
  unsigned long long c = 0;
  const size_t nv = n / 8, stride = (size_t)gridDim.x * blockDim.x;
  const size_t t0 = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (size_t v = t0; v < nv; v += stride) c += nonfinite8<T>(x + v * 8);
  if (t0 == 0)  // ragged tail (n % 8 elements)
    for (size_t e = nv * 8; e < n; ++e) {
      uint32_t u;
      if constexpr (sizeof(T) == 2) u = (uint32_t)((const uint16_t*)x)[e] << 16;
      else u = ((const uint32_t*)x)[e];
      c += (u & 0x7f800000u) == 0x7f800000u;
    }
  for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, 64);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) part[blockIdx.x] = sh[0] + sh[1] + sh[2] + sh[3];
}

__global__ void nonfinite_pass2_k(const unsigned long long* part, int nblk, unsigned long long* out) {
  if (threadIdx.x == 0) {
    unsigned long long c = 0;
    for (int b = 0; b < nblk; ++b) c += part[b];
    *out = c;
  }
}

int count_nonfinite(const void* x, size_t n, int dt, unsigned long long* part, unsigned long long* out_dev,
                    hipStream_t s) {
  if (!x || n == 0) { set_error("count_nonfinite: empty or null vector"); return 1; }
  if (((uintptr_t)x & 15) != 0) { set_error("count_nonfinite: vector must be 16-byte aligned"); return 1; }
  const size_t nv = n / 8;
  const unsigned grid = (unsigned)std::max<size_t>(1, std::min<size_t>((nv + 255) / 256, CMP_BLOCKS));
  if (dt == BF16) hipLaunchKernelGGL(nonfinite_pass1_k<uint16_t>, dim3(grid), dim3(256), 0, s, (const uint16_t*)x, n, part);
  else hipLaunchKernelGGL(nonfinite_pass1_k<float>, dim3(grid), dim3(256), 0, s, (const float*)x, n, part);
  LAUNCH_OK("count_nonfinite_pass1");
  hipLaunchKernelGGL(nonfinite_pass2_k, dim3(1), dim3(64), 0, s, part, (int)grid, out_dev);
  LAUNCH_OK("count_nonfinite_pass2");
  return 0;
}

// ================================================================ GRPO window
// Phase 2 (upstream gradients of the PPO-clipped GRPO loss through the
// rectified-flow Euler step) fused with Phase 3 (composites), three launches:
//   pass 1: per sample b and step j, sq[j][b] = |z_{j+1} - z_j - dt_j v_j|^2
//           in fp64 (block partials, fixed order);
//   coef:   log pi_j = -sq / (2 sigma_j^2) - n log(sqrt(2 pi) sigma_j),
//           rho_j = exp(log pi_j - log pi_old_j), A = clamp(A_b, +-adv_clip),
//           dL/drho = 0 if the clipped PPO term is strictly the larger, else
//           -A / W, and coef[j][b] = dL/drho * rho_j * dt_j / sigma_j^2;
//   pass 2: r_j = z_{j+1} - z_j - dt_j v_j (fp32) and either the composites
//           s_base = sum_j (1 - alpha_j) coef_j r_j, s_corr = sum_j alpha_j
//           coef_j r_j (one rounding on store) or the W gradients coef_j r_j.
// s_j = coef_j r_j never reaches memory in the composite mode.  HBM traffic
// per element: (2W + 1) reads in each pass, plus 2 (or W) writes.
// pass-1 blocks per sample: enough blocks in total to stream at full HBM
// bandwidth, while the W x B x blocks partials stay within a fixed buffer
constexpr int GRPO_PART_MAX = 32768;
static int grpo_blocks(int W, int B) { return std::max(1, std::min(2048 / B + 1, GRPO_PART_MAX / (W * B))); }
size_t grpo_part_doubles(int W, int B) { (void)W; (void)B; return GRPO_PART_MAX; }

template <typename T>
__device__ __forceinline__ size_t grpo_elem(const GrpoArgs& a, int b, size_t i) {
  return i < a.len0 ? (size_t)b * a.len0 + i : a.split + (size_t)b * a.len1 + (i - a.len0);
}
// element i of sample b inside v_j, which holds samples vk .. vk+B-1 of a
// batch-vb array in the same layout (an endpoint pair, a batch of middle steps)
__device__ __forceinline__ size_t grpo_velem(const GrpoArgs& a, int j, int b, size_t i) {
  const size_t bb = (size_t)a.vk[j] + b;
  return i < a.len0 ? bb * a.len0 + i : (size_t)a.vb[j] * a.len0 + bb * a.len1 + (i - a.len0);
}

template <typename T, int W>
__global__ __launch_bounds__(256) void grpo_sq_k(GrpoArgs a, double* part) {
  __shared__ double sh[4][W];
  const int b = blockIdx.y;
  const size_t per = (a.len0 + a.len1) / 8;  // vectors per sample
  double acc[W];
#pragma unroll
  for (int j = 0; j < W; ++j) acc[j] = 0.0;
  for (size_t v = (size_t)blockIdx.x * blockDim.x + threadIdx.x; v < per; v += (size_t)gridDim.x * blockDim.x) {
    const size_t e = grpo_elem<T>(a, b, v * 8);
    float zc[8];
    load8f<T>((const T*)a.z[0] + e, zc);
#pragma unroll
    for (int j = 0; j < W; ++j) {
      float zn[8], vv[8];
      load8f<T>((const T*)a.z[j + 1] + e, zn);
      load8f<T>((const T*)a.v[j] + grpo_velem(a, j, b, v * 8), vv);
      const double dtj = a.dts[j];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const double r = ((double)zn[q] - (double)zc[q]) - dtj * (double)vv[q];
        acc[j] = fma(r, r, acc[j]);
        zc[q] = zn[q];
      }
    }
  }
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
#pragma unroll
  for (int j = 0; j < W; ++j) {
    double x = acc[j];
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
    if (lane == 0) sh[wv][j] = x;
  }
  __syncthreads();
  if (threadIdx.x < W)
    part[((size_t)threadIdx.x * a.B + b) * gridDim.x + blockIdx.x] =
        sh[0][threadIdx.x] + sh[1][threadIdx.x] + sh[2][threadIdx.x] + sh[3][threadIdx.x];
}

// one block per (j, b): the block partials summed in a fixed order (strided
// per thread, then a fixed shuffle and LDS tree), then the closed-form scalars
__global__ __launch_bounds__(256) void grpo_coef_k(GrpoArgs a, const double* part, int nblk, float* coef,
                                                   double* stats) {
  __shared__ double sh[4];
  const int k = blockIdx.x;  // k = j * B + b
  const int j = k / a.B, b = k % a.B;
  double x = 0.0;
  for (int i = threadIdx.x; i < nblk; i += blockDim.x) x += part[(size_t)k * nblk + i];
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = x;
  __syncthreads();
  if (threadIdx.x != 0) return;
  const double sq = (sh[0] + sh[1]) + (sh[2] + sh[3]);
  const double sg = a.sigma[j];
  const double n = (double)(a.len0 + a.len1);
  const double lp = -sq / (2.0 * sg * sg) - n * log(sqrt(2.0 * M_PI) * sg);
  const double rho = exp(lp - a.logp_old[k]);
  const double A = fmin(fmax((double)a.adv[b], -(double)a.adv_clip), (double)a.adv_clip);
  const double unc = -A * rho;
  const double clp = -A * fmin(fmax(rho, 1.0 - (double)a.eps), 1.0 + (double)a.eps);
  const double dl = clp > unc ? 0.0 : -A / a.W;
  coef[k] = (float)(dl * rho * a.dts[j] / (sg * sg));
  if (stats) {
    stats[3 * k] = lp;
    stats[3 * k + 1] = rho;
    stats[3 * k + 2] = fmax(unc, clp) / a.W;
  }
}

template <typename T>
__device__ __forceinline__ void store8f(T* p, const float* x) {
  if constexpr (sizeof(T) == 2) {
    uint4 u;
    u.x = f2bf(x[0]) | ((uint32_t)f2bf(x[1]) << 16); u.y = f2bf(x[2]) | ((uint32_t)f2bf(x[3]) << 16);
    u.z = f2bf(x[4]) | ((uint32_t)f2bf(x[5]) << 16); u.w = f2bf(x[6]) | ((uint32_t)f2bf(x[7]) << 16);
    *(uint4*)p = u;
  } else {
    *(float4*)p = make_float4(x[0], x[1], x[2], x[3]);
    *(float4*)(p + 4) = make_float4(x[4], x[5], x[6], x[7]);
  }
}

template <typename T, int W>
__global__ __launch_bounds__(256) void grpo_out_k(GrpoArgs a, const float* coef) {
  const size_t nv = a.n / 8;
  for (size_t v = (size_t)blockIdx.x * blockDim.x + threadIdx.x; v < nv; v += (size_t)gridDim.x * blockDim.x) {
    const size_t e = v * 8;
    const int b = (int)(e < a.split ? e / a.len0 : (e - a.split) / a.len1);
    const size_t i = e < a.split ? e - (size_t)b * a.len0 : a.len0 + (e - a.split) - (size_t)b * a.len1;
    float zc[8], sb[8], sc[8];
    load8f<T>((const T*)a.z[0] + e, zc);
#pragma unroll
    for (int q = 0; q < 8; ++q) sb[q] = sc[q] = 0.f;
#pragma unroll
    for (int j = 0; j < W; ++j) {
      float zn[8], vv[8], sj[8];
      load8f<T>((const T*)a.z[j + 1] + e, zn);
      load8f<T>((const T*)a.v[j] + grpo_velem(a, j, b, i), vv);
      const float c = coef[j * a.B + b], dtj = (float)a.dts[j];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        sj[q] = c * ((zn[q] - zc[q]) - dtj * vv[q]);
        zc[q] = zn[q];
      }
      if (a.mode == 1) {
        store8f<T>((T*)a.s_out[j] + e, sj);
      } else {
#pragma unroll
        for (int q = 0; q < 8; ++q) { sb[q] = fmaf(a.wb[j], sj[q], sb[q]); sc[q] = fmaf(a.wc[j], sj[q], sc[q]); }
      }
    }
    if (a.mode == 0) {
      if (e < a.osplit) { store8f<T>((T*)a.base0 + e, sb); store8f<T>((T*)a.corr0 + e, sc); }
      else { store8f<T>((T*)a.base1 + (e - a.osplit), sb); store8f<T>((T*)a.corr1 + (e - a.osplit), sc); }
    }
  }
}

// The three kernels of a window; under timing each is its own record (work in
// bytes: pass 1 reads z_0..z_W and the v_j, the closed-form scalars move
// nothing of size, pass 2 reads them again and writes the composites or s_j).
template <typename T, int W>
static void grpo_launch(const GrpoArgs& a, double* part, float* coef, double* stats, hipStream_t s) {
  const int ch = grpo_blocks(a.W, a.B);
  const double es = dsize(a.dt), pass = (double)a.n * es * (2 * a.W + 1);
  int pi = prof_begin(PROF_UPSTREAM);
  launch(grpo_sq_k<T, W>, dim3(ch, a.B), dim3(256), 0u, s, a, part);
  prof_end(pi, pass);
  pi = prof_begin(PROF_UPSTREAM);
  launch(grpo_coef_k, dim3(a.W * a.B), dim3(256), 0u, s, a, part, ch, coef, stats);
  prof_end(pi, 0.0);
  const size_t nv = a.n / 8;
  const unsigned grid = (unsigned)std::max<size_t>(1, std::min<size_t>((nv + 255) / 256, 256 * 16));
  pi = prof_begin(PROF_UPSTREAM);
  launch(grpo_out_k<T, W>, dim3(grid), dim3(256), 0u, s, a, coef);
  prof_end(pi, pass + (double)a.n * es * (a.mode == 1 ? a.W : 2));
}

int grpo_window(const GrpoArgs& a, double* part, float* coef, double* stats, hipStream_t s) {
  if (a.W < 2 || a.W > GRPO_MAX_W || a.B < 1) { set_error("grpo_window: W must be 2..16, B >= 1"); return 1; }
  if (a.len0 % 8 || a.len1 % 8 || a.split % 8 || a.osplit % 8 || a.len0 + a.len1 == 0) {
    set_error("grpo_window: per-sample segments must be multiples of 8 elements");
    return 4;
  }
#define GRPO_W(T, w) case w: grpo_launch<T, w>(a, part, coef, stats, s); break;
  if (a.dt == BF16) {
    switch (a.W) { GRPO_W(uint16_t, 2) GRPO_W(uint16_t, 3) GRPO_W(uint16_t, 4) GRPO_W(uint16_t, 5) GRPO_W(uint16_t, 6)
                   GRPO_W(uint16_t, 7) GRPO_W(uint16_t, 8) GRPO_W(uint16_t, 10) GRPO_W(uint16_t, 12)
                   GRPO_W(uint16_t, 16)
      default: set_error("grpo_window: W must be one of 2..8, 10, 12, 16"); return 4; }
  } else {
    switch (a.W) { GRPO_W(float, 2) GRPO_W(float, 3) GRPO_W(float, 4) GRPO_W(float, 5) GRPO_W(float, 6)
                   GRPO_W(float, 7) GRPO_W(float, 8) GRPO_W(float, 10) GRPO_W(float, 12) GRPO_W(float, 16)
      default: set_error("grpo_window: W must be one of 2..8, 10, 12, 16"); return 4; }
  }
#undef GRPO_W
  LAUNCH_OK("grpo_window");
  return 0;
}

}  // namespace jg
