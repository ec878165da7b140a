// Reference-precision attention on the vector ALUs: online-softmax forward and
// the two-kernel backward (dK/dV over query tiles, dQ over key tiles), fp32
// arithmetic for fp32 or bf16 storage, any head dim up to 128 (multiple of 4).
// Four threads share one query (or key) row, each owning Dh/4 dims; K/V (or
// Q/dO) tiles are staged in LDS.  The bf16 hot path uses the MFMA kernels in
// attention_mfma.hip; this file serves the fp32 path and odd shapes.
#include "attention.h"

namespace jg {

__device__ inline int row_of_tok(const RowMap& rm, int b, int j) {
  return j < rm.nt ? b * rm.nt + j : rm.B * rm.nt + b * rm.ni + (j - rm.nt);
}

constexpr int AV_Q = 64;  // rows per block (4 threads each)
constexpr int AV_K = 64;  // staged rows per tile

template <int DH, typename T>
__global__ __launch_bounds__(256) void attn_fwd_valu_k(AttnFwd a) {
  constexpr int DPT = DH / 4;
  __shared__ float Ks[AV_K][DH];
  __shared__ float Vs[AV_K][DH];
  const int bh = blockIdx.y, b = bh / a.H, h = bh % a.H;
  const int qi = threadIdx.x >> 2, t = threadIdx.x & 3;
  const int j = blockIdx.x * AV_Q + qi;
  const bool valid = j < a.N;
  const size_t base = (size_t)bh * a.N * DH;
  const T* Q = (const T*)a.Q;
  const T* K = (const T*)a.K;
  const T* V = (const T*)a.V;
  const float scale = rsqrtf((float)DH);
  float q[DPT], acc[DPT];
#pragma unroll
  for (int d = 0; d < DPT; ++d) {
    q[d] = valid ? ldf(Q, base + (size_t)j * DH + t * DPT + d) * scale : 0.f;
    acc[d] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int k0 = 0; k0 < a.N; k0 += AV_K) {
    __syncthreads();
    for (int i = threadIdx.x; i < AV_K * DH; i += 256) {
      const int kk = i / DH, d = i % DH;
      const bool in = k0 + kk < a.N;
      Ks[kk][d] = in ? ldf(K, base + (size_t)(k0 + kk) * DH + d) : 0.f;
      Vs[kk][d] = in ? ldf(V, base + (size_t)(k0 + kk) * DH + d) : 0.f;
    }
    __syncthreads();
    const int kn = min(AV_K, a.N - k0);
    for (int kk = 0; kk < kn; ++kk) {
      float s = 0.f;
#pragma unroll
      for (int d = 0; d < DPT; ++d) s = fmaf(q[d], Ks[kk][t * DPT + d], s);
      s += __shfl_xor(s, 1, 64);
      s += __shfl_xor(s, 2, 64);
      const float mn = fmaxf(m, s);
      const float corr = __expf(m - mn), p = __expf(s - mn);
      l = l * corr + p;
#pragma unroll
      for (int d = 0; d < DPT; ++d) acc[d] = fmaf(p, Vs[kk][t * DPT + d], acc[d] * corr);
      m = mn;
    }
  }
  if (!valid) return;
  T* O = (T*)a.O;
  const size_t orow = (size_t)row_of_tok(a.rm, b, j) * a.ld_o + h * DH + t * DPT;
  const float inv = 1.f / l;
#pragma unroll
  for (int d = 0; d < DPT; ++d) stf(O, orow + d, acc[d] * inv);
  if (t == 0) a.lse[(size_t)bh * a.N + j] = m + logf(l);
}

template <typename T>
__global__ void attn_delta_k(AttnBwd a) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t n = (size_t)a.B * a.H * a.N;
  if (i >= n) return;
  const int j = (int)(i % a.N);
  const int bh = (int)(i / a.N), b = bh / a.H, h = bh % a.H;
  const size_t r = row_of_tok(a.rm, b, j);
  const T* O = (const T*)a.O;
  const T* dO = (const T*)a.dO;
  float s = 0.f;
  for (int d = 0; d < a.Dh; ++d) s = fmaf(ldf(O, r * a.ld_o + h * a.Dh + d), ldf(dO, r * a.ld_do + h * a.Dh + d), s);
  a.delta[i] = s;
}

template <int DH, typename T, typename TD>
__global__ __launch_bounds__(256) void attn_bwd_kv_valu_k(AttnBwd a) {
  constexpr int DPT = DH / 4;
  __shared__ float Qs[AV_K][DH];
  __shared__ float dOs[AV_K][DH];
  __shared__ float Ls[AV_K], Ds[AV_K];
  const int bh = blockIdx.y, b = bh / a.H, h = bh % a.H;
  const int ki = threadIdx.x >> 2, t = threadIdx.x & 3;
  const int j = blockIdx.x * AV_Q + ki;
  const bool valid = j < a.N;
  const size_t base = (size_t)bh * a.N * DH;
  const T* Q = (const T*)a.Q;
  const T* K = (const T*)a.K;
  const T* V = (const T*)a.V;
  const T* dO = (const T*)a.dO;
  const float scale = rsqrtf((float)DH);
  float k[DPT], v[DPT], dk[DPT], dv[DPT];
#pragma unroll
  for (int d = 0; d < DPT; ++d) {
    k[d] = valid ? ldf(K, base + (size_t)j * DH + t * DPT + d) : 0.f;
    v[d] = valid ? ldf(V, base + (size_t)j * DH + t * DPT + d) : 0.f;
    dk[d] = dv[d] = 0.f;
  }
  for (int i0 = 0; i0 < a.N; i0 += AV_K) {
    __syncthreads();
    for (int e = threadIdx.x; e < AV_K * DH; e += 256) {
      const int ii = e / DH, d = e % DH;
      const bool in = i0 + ii < a.N;
      Qs[ii][d] = in ? ldf(Q, base + (size_t)(i0 + ii) * DH + d) : 0.f;
      dOs[ii][d] = in ? ldf(dO, (size_t)row_of_tok(a.rm, b, i0 + ii) * a.ld_do + h * DH + d) : 0.f;
    }
    for (int e = threadIdx.x; e < AV_K; e += 256) {
      const bool in = i0 + e < a.N;
      Ls[e] = in ? a.lse[(size_t)bh * a.N + i0 + e] : 0.f;
      Ds[e] = in ? a.delta[(size_t)bh * a.N + i0 + e] : 0.f;
    }
    __syncthreads();
    const int qn = min(AV_K, a.N - i0);
    for (int ii = 0; ii < qn; ++ii) {
      float s = 0.f, dp = 0.f;
#pragma unroll
      for (int d = 0; d < DPT; ++d) {
        s = fmaf(Qs[ii][t * DPT + d], k[d], s);
        dp = fmaf(dOs[ii][t * DPT + d], v[d], dp);
      }
      s += __shfl_xor(s, 1, 64);
      s += __shfl_xor(s, 2, 64);
      dp += __shfl_xor(dp, 1, 64);
      dp += __shfl_xor(dp, 2, 64);
      const float p = __expf(s * scale - Ls[ii]);
      const float ds = p * (dp - Ds[ii]) * scale;
#pragma unroll
      for (int d = 0; d < DPT; ++d) {
        dv[d] = fmaf(p, dOs[ii][t * DPT + d], dv[d]);
        dk[d] = fmaf(ds, Qs[ii][t * DPT + d], dk[d]);
      }
    }
  }
  if (!valid) return;
#pragma unroll
  for (int d = 0; d < DPT; ++d) {
    stf((TD*)a.dK, base + (size_t)j * DH + t * DPT + d, dk[d]);
    stf((TD*)a.dV, base + (size_t)j * DH + t * DPT + d, dv[d]);
  }
}

template <int DH, typename T, typename TD>
__global__ __launch_bounds__(256) void attn_bwd_q_valu_k(AttnBwd a) {
  constexpr int DPT = DH / 4;
  __shared__ float Ks[AV_K][DH];
  __shared__ float Vs[AV_K][DH];
  const int bh = blockIdx.y, b = bh / a.H, h = bh % a.H;
  const int qi = threadIdx.x >> 2, t = threadIdx.x & 3;
  const int j = blockIdx.x * AV_Q + qi;
  const bool valid = j < a.N;
  const size_t base = (size_t)bh * a.N * DH;
  const T* Q = (const T*)a.Q;
  const T* K = (const T*)a.K;
  const T* V = (const T*)a.V;
  const T* dO = (const T*)a.dO;
  const float scale = rsqrtf((float)DH);
  float q[DPT], g[DPT], dq[DPT];
  const size_t r = valid ? (size_t)row_of_tok(a.rm, b, j) : 0;
#pragma unroll
  for (int d = 0; d < DPT; ++d) {
    q[d] = valid ? ldf(Q, base + (size_t)j * DH + t * DPT + d) : 0.f;
    g[d] = valid ? ldf(dO, r * a.ld_do + h * DH + t * DPT + d) : 0.f;
    dq[d] = 0.f;
  }
  const float L = valid ? a.lse[(size_t)bh * a.N + j] : 0.f;
  const float Dl = valid ? a.delta[(size_t)bh * a.N + j] : 0.f;
  for (int k0 = 0; k0 < a.N; k0 += AV_K) {
    __syncthreads();
    for (int e = threadIdx.x; e < AV_K * DH; e += 256) {
      const int kk = e / DH, d = e % DH;
      const bool in = k0 + kk < a.N;
      Ks[kk][d] = in ? ldf(K, base + (size_t)(k0 + kk) * DH + d) : 0.f;
      Vs[kk][d] = in ? ldf(V, base + (size_t)(k0 + kk) * DH + d) : 0.f;
    }
    __syncthreads();
    const int kn = min(AV_K, a.N - k0);
    for (int kk = 0; kk < kn; ++kk) {
      float s = 0.f, dp = 0.f;
#pragma unroll
      for (int d = 0; d < DPT; ++d) {
        s = fmaf(q[d], Ks[kk][t * DPT + d], s);
        dp = fmaf(g[d], Vs[kk][t * DPT + d], dp);
      }
      s += __shfl_xor(s, 1, 64);
      s += __shfl_xor(s, 2, 64);
      dp += __shfl_xor(dp, 1, 64);
      dp += __shfl_xor(dp, 2, 64);
      const float p = __expf(s * scale - L);
      const float ds = p * (dp - Dl) * scale;
#pragma unroll
      for (int d = 0; d < DPT; ++d) dq[d] = fmaf(ds, Ks[kk][t * DPT + d], dq[d]);
    }
  }
  if (!valid) return;
#pragma unroll
  for (int d = 0; d < DPT; ++d) stf((TD*)a.dQ, base + (size_t)j * DH + t * DPT + d, dq[d]);
}

// ------------------------------------------------------------------ launch
template <int DH>
static void fwd_valu(const AttnFwd& a, hipStream_t s) {
  dim3 grid((a.N + AV_Q - 1) / AV_Q, a.B * a.H);
  if (a.dt == BF16) hipLaunchKernelGGL((attn_fwd_valu_k<DH, uint16_t>), grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL((attn_fwd_valu_k<DH, float>), grid, dim3(256), 0, s, a);
}

template <int DH, typename T, typename TD>
static void bwd_valu_t(const AttnBwd& a, hipStream_t s) {
  dim3 grid((a.N + AV_Q - 1) / AV_Q, a.B * a.H);
  hipLaunchKernelGGL((attn_bwd_kv_valu_k<DH, T, TD>), grid, dim3(256), 0, s, a);
  hipLaunchKernelGGL((attn_bwd_q_valu_k<DH, T, TD>), grid, dim3(256), 0, s, a);
}

template <int DH>
static void bwd_valu(const AttnBwd& a, hipStream_t s) {
  if (a.dt == BF16 && a.dt_d == BF16) bwd_valu_t<DH, uint16_t, uint16_t>(a, s);
  else if (a.dt == BF16) bwd_valu_t<DH, uint16_t, float>(a, s);
  else if (a.dt_d == BF16) bwd_valu_t<DH, float, uint16_t>(a, s);
  else bwd_valu_t<DH, float, float>(a, s);
}

int attention_fwd_mfma(const AttnFwd& a, hipStream_t s);  // attention_mfma.hip; returns -1 if not applicable
int attention_bwd_mfma(const AttnBwd& a, hipStream_t s);

int attention_fwd(const AttnFwd& a, hipStream_t s) {
  if (a.N <= 0 || a.B <= 0 || a.H <= 0) { set_error("attention_fwd: empty problem"); return 1; }
  const int rc = attention_fwd_mfma(a, s);
  if (rc >= 0) return rc;
  switch (a.Dh) {
    case 16: fwd_valu<16>(a, s); break;
    case 32: fwd_valu<32>(a, s); break;
    case 64: fwd_valu<64>(a, s); break;
    case 128: fwd_valu<128>(a, s); break;
    default: set_error("attention_fwd: head_dim must be 16, 32, 64 or 128"); return 4;
  }
  JG_CHECK_LAUNCH("attention_fwd_valu");
  return 0;
}

int attention_bwd(const AttnBwd& a, hipStream_t s) {
  if (a.N <= 0 || a.B <= 0 || a.H <= 0) { set_error("attention_bwd: empty problem"); return 1; }
  const int rc = attention_bwd_mfma(a, s);
  if (rc >= 0) return rc;
  const size_t n = (size_t)a.B * a.H * a.N;
  if (a.dt == BF16) hipLaunchKernelGGL(attn_delta_k<uint16_t>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a);
  else hipLaunchKernelGGL(attn_delta_k<float>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a);
  JG_CHECK_LAUNCH("attention_delta");
  switch (a.Dh) {
    case 16: bwd_valu<16>(a, s); break;
    case 32: bwd_valu<32>(a, s); break;
    case 64: bwd_valu<64>(a, s); break;
    case 128: bwd_valu<128>(a, s); break;
    default: set_error("attention_bwd: head_dim must be 16, 32, 64 or 128"); return 4;
  }
  JG_CHECK_LAUNCH("attention_bwd_valu");
  return 0;
}

}  // namespace jg
