// Flash attention forward and backward on gfx950 MFMA (bf16 in, fp32
// accumulation), head dim 128.
//
// Layout trick: every score tile is computed in the orientation whose MFMA
// accumulator can feed the next MFMA directly as its "B" operand.  With
// v_mfma_f32_32x32x16_bf16 a lane holds one column j (lane % 32) of the 32x32
// accumulator and 16 rows 8*(e/4) + 4*(lane/32) + e%4.  Taking the contraction
// slots of the next product as those same rows, the 8 fp32 values
// e = 8c .. 8c+7 of a lane are exactly its bf16 B fragment for 16-row block c,
// provided the A operand is read with the same row order (two 8-byte LDS
// reads at rows 16c + 4h and 16c + 8 + 4h).  Hence:
//   forward:  S^T = K Q^T, O^T += V^T P^T   (query = lane column: softmax
//             statistics and the rescale of O stay inside the lane)
//   dK/dV:    S = Q K^T, dP = dO V^T, dV^T += dO^T P, dK^T += Q^T dS
//   dQ:       S^T = K Q^T, dP^T = V dO^T, dQ^T += K^T dS^T
// Softmax works in the log2 domain with the hardware exp2; the stored
// log-sum-exp is in natural-log units of the scaled scores (shared with the
// VALU kernels).  Ragged sequence lengths are masked (keys >= N get P = 0,
// padded queries are not written).
#include "attention.h"
#include "prof.h"
#include <type_traits>

namespace jg {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

constexpr int DH = 128;
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

__device__ inline int row_of_tok_m(const RowMap& rm, int b, int j) {
  return j < rm.nt ? b * rm.nt + j : rm.B * rm.nt + b * rm.ni + (j - rm.nt);
}

__device__ inline f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ inline f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}

// 16-byte read of 8 bf16 at p (LDS or global)
__device__ inline bf16x8 ld8(const uint16_t* p) { return __builtin_bit_cast(bf16x8, *(const u32x4*)p); }
// two 8-byte reads at p and p + 8 elements (rows 16c+4h.. and 16c+8+4h..)
__device__ inline bf16x8 ld4x2(const uint16_t* p) {
  const u32x2 a = *(const u32x2*)p, b = *(const u32x2*)(p + 8);
  u32x4 r = {a[0], a[1], b[0], b[1]};
  return __builtin_bit_cast(bf16x8, r);
}
// accumulator values e = 8c .. 8c+7 as a bf16 B fragment
__device__ inline bf16x8 pack8(const f32x16& v, int c) {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = (__bf16)v[8 * c + i];
  return r;
}

// Stage a T x 128 tile (rows r0.., head-major rows of length 128) into LDS
// S[r][d] (stride DS); rows >= nrows are zero.
template <int T, int DS>
__device__ inline void stage_rows(uint16_t* S, const uint16_t* G, int r0, int nrows) {
  for (int v = threadIdx.x; v < T * (DH / 8); v += 256) {
    const int r = v / (DH / 8), c = v % (DH / 8);
    u32x4 x = {0u, 0u, 0u, 0u};
    if (r0 + r < nrows) x = *(const u32x4*)(G + (size_t)(r0 + r) * DH + c * 8);
    *(u32x4*)(S + r * DS + c * 8) = x;
  }
}
// Same tile transposed: S[d][r] (stride TS)
template <int T, int TS>
__device__ inline void stage_rows_t(uint16_t* S, const uint16_t* G, int r0, int nrows) {
  for (int v = threadIdx.x; v < T * (DH / 8); v += 256) {
    const int r = v % T, c = v / T;
    u32x4 x = {0u, 0u, 0u, 0u};
    if (r0 + r < nrows) x = *(const u32x4*)(G + (size_t)(r0 + r) * DH + c * 8);
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      S[(c * 8 + 2 * w) * TS + r] = (uint16_t)(x[w] & 0xffffu);
      S[(c * 8 + 2 * w + 1) * TS + r] = (uint16_t)(x[w] >> 16);
    }
  }
}
// Token-major rows (the attention output layout): row j of sample b at
// rows row_of_tok(b, j), columns h*128 ..
template <int T, int DS>
__device__ inline void stage_tok(uint16_t* S, const uint16_t* G, int ld, const RowMap& rm, int b, int h, int j0,
                                 int N) {
  for (int v = threadIdx.x; v < T * (DH / 8); v += 256) {
    const int r = v / (DH / 8), c = v % (DH / 8);
    u32x4 x = {0u, 0u, 0u, 0u};
    if (j0 + r < N) x = *(const u32x4*)(G + (size_t)row_of_tok_m(rm, b, j0 + r) * ld + h * DH + c * 8);
    *(u32x4*)(S + r * DS + c * 8) = x;
  }
}
template <int T, int TS>
__device__ inline void stage_tok_t(uint16_t* S, const uint16_t* G, int ld, const RowMap& rm, int b, int h, int j0,
                                   int N) {
  for (int v = threadIdx.x; v < T * (DH / 8); v += 256) {
    const int r = v % T, c = v / T;
    u32x4 x = {0u, 0u, 0u, 0u};
    if (j0 + r < N) x = *(const u32x4*)(G + (size_t)row_of_tok_m(rm, b, j0 + r) * ld + h * DH + c * 8);
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      S[(c * 8 + 2 * w) * TS + r] = (uint16_t)(x[w] & 0xffffu);
      S[(c * 8 + 2 * w + 1) * TS + r] = (uint16_t)(x[w] >> 16);
    }
  }
}

// Register-staged tile: T rows x 128 columns, fetched as 8x8 element blocks
// (one block per participating thread: 8 x 16-byte loads, one per row) so
// that the same registers can be written to LDS both as rows (S[r][d]) and,
// after an in-register 8x8 transpose, as columns (S^T[d][r]).  `load` is
// issued one tile ahead of its use; `commit` writes the LDS copies.
template <int T>
struct Tile8 {
  static constexpr int NBLK = (T / 8) * (DH / 8);  // blocks per tile
  u32x4 r[8];
  int rb, db;
  bool on;
  __device__ inline void init(int slot) {  // slot in [0, NBLK) or -1
    on = slot >= 0 && slot < NBLK;
    db = on ? slot % (DH / 8) : 0;
    rb = on ? slot / (DH / 8) : 0;
  }
  // rowptr(i) = pointer to row i (or nullptr when the row is out of range)
  template <class RowPtr>
  __device__ inline void load(RowPtr rowptr, int r0) {
    if (!on) return;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const uint16_t* p = rowptr(r0 + rb * 8 + k);
      r[k] = p ? *(const u32x4*)(p + db * 8) : u32x4{0u, 0u, 0u, 0u};
    }
  }
  template <int DS>
  __device__ inline void commit_rows(uint16_t* S) const {
    if (!on) return;
#pragma unroll
    for (int k = 0; k < 8; ++k) *(u32x4*)(S + (rb * 8 + k) * DS + db * 8) = r[k];
  }
  template <int TS>
  __device__ inline void commit_cols(uint16_t* S) const {
    if (!on) return;
    // word w of row m of the transposed block = element (r = 2w, m) | (r = 2w+1, m) << 16
#pragma unroll
    for (int mw = 0; mw < 4; ++mw) {
      u32x4 lo, hi;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const unsigned a = r[2 * w][mw], c = r[2 * w + 1][mw];
        lo[w] = (a & 0xffffu) | (c << 16);
        hi[w] = (a >> 16) | (c & 0xffff0000u);
      }
      *(u32x4*)(S + (db * 8 + 2 * mw) * TS + rb * 8) = lo;
      *(u32x4*)(S + (db * 8 + 2 * mw + 1) * TS + rb * 8) = hi;
    }
  }
};

// ============================================================== forward
constexpr int F_QB = 128, F_KT = 64;
constexpr int F_KS = DH + 8;    // K tile row stride
constexpr int F_VS = F_KT + 8;  // V^T tile row stride

__global__ __launch_bounds__(256) void attn_fwd_mfma_k(AttnFwd a) {
  __shared__ __attribute__((aligned(16))) uint16_t Ks[F_KT * F_KS];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[DH * F_VS];
  const int bh = blockIdx.y, b = bh / a.H, hd = bh % a.H;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, h = lane >> 5, c32 = lane & 31;
  const int q = blockIdx.x * F_QB + w * 32 + c32;  // this lane's query
  const size_t base = (size_t)bh * a.N * DH;
  const uint16_t* Q = (const uint16_t*)a.Q + base;
  const uint16_t* K = (const uint16_t*)a.K + base;
  const uint16_t* V = (const uint16_t*)a.V + base;
  const float sc = rsqrtf((float)DH) * LOG2E;
  const int N = a.N;

  // threads [0, 128) stage K blocks, [128, 256) V blocks (64 keys x 128 = 128 blocks each)
  Tile8<F_KT> tk;
  const bool isk = threadIdx.x < 128;
  tk.init(isk ? (int)threadIdx.x : (int)threadIdx.x - 128);
  const uint16_t* src = isk ? K : V;
  auto rows = [&](int i) -> const uint16_t* { return i < N ? src + (size_t)i * DH : nullptr; };

  bf16x8 qf[8];
#pragma unroll
  for (int kb = 0; kb < 8; ++kb) {
    if (q < N) qf[kb] = ld8(Q + (size_t)q * DH + kb * 16 + h * 8);
    else qf[kb] = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
  }
  f32x16 o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = zero16();
  float m = -INFINITY, l = 0.f;

  tk.load(rows, 0);
  for (int k0 = 0; k0 < N; k0 += F_KT) {
    __syncthreads();  // everyone is done reading the previous tile
    if (isk) tk.commit_rows<F_KS>(Ks);
    else tk.commit_cols<F_VS>(Vt);
    __syncthreads();
    if (k0 + F_KT < N) tk.load(rows, k0 + F_KT);  // lands during this tile's MFMAs
    f32x16 st[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      st[t] = zero16();
#pragma unroll
      for (int kb = 0; kb < 8; ++kb) st[t] = mfma(ld8(Ks + (32 * t + c32) * F_KS + kb * 16 + h * 8), qf[kb], st[t]);
    }
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int key = k0 + 32 * t + 8 * (e >> 2) + 4 * h + (e & 3);
        const float sv = key < N ? st[t][e] * sc : -INFINITY;
        st[t][e] = sv;
        mx = fmaxf(mx, sv);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float mn = fmaxf(m, mx);
    const float corr = __builtin_amdgcn_exp2f(m - mn);
    float ls = 0.f;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float p = __builtin_amdgcn_exp2f(st[t][e] - mn);
        st[t][e] = p;
        ls += p;
      }
    l = l * corr + ls;
    m = mn;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[i][e] *= corr;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const bf16x8 pb = pack8(st[c >> 1], c & 1);
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) o[dt] = mfma(ld4x2(Vt + (32 * dt + c32) * F_VS + 16 * c + 4 * h), pb, o[dt]);
    }
  }
  l += __shfl_xor(l, 32, 64);
  if (q >= N) return;
  const float inv = 1.f / l;
  uint16_t* O = (uint16_t*)a.O + (size_t)row_of_tok_m(a.rm, b, q) * a.ld_o + hd * DH;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x4 v;
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = (__bf16)(o[dt][4 * g + i] * inv);
      *(bf16x4*)(O + 32 * dt + 8 * g + 4 * h) = v;
    }
  if (h == 0) a.lse[(size_t)bh * N + q] = (m + __log2f(l)) * LN2;
}

// ============================================================== delta
// delta[b][h][j] = sum_d dO[j][h*128+d] * O[j][h*128+d]; one wave per row,
// 16 lanes per head, 16-byte loads.
__global__ __launch_bounds__(256) void attn_delta_mfma_k(AttnBwd a) {
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int rows = a.rm.rows();
  if (r >= rows) return;
  const int bt = a.rm.B * a.rm.nt;
  int b, j;
  if (r < bt) { b = r / a.rm.nt; j = r % a.rm.nt; }
  else { b = (r - bt) / a.rm.ni; j = a.rm.nt + (r - bt) % a.rm.ni; }
  const uint16_t* O = (const uint16_t*)a.O + (size_t)r * a.ld_o;
  const uint16_t* G = (const uint16_t*)a.dO + (size_t)r * a.ld_do;
  const int D = a.H * DH;
  for (int c0 = 0; c0 < D; c0 += 512) {
    const int c = c0 + lane * 8;
    float s = 0.f;
    if (c < D) {
      const u32x4 x = *(const u32x4*)(O + c), y = *(const u32x4*)(G + c);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        s = fmaf(bf2f(x[w] & 0xffffu), bf2f(y[w] & 0xffffu), s);
        s = fmaf(bf2f(x[w] >> 16), bf2f(y[w] >> 16), s);
      }
    }
    s += __shfl_xor(s, 1, 64);
    s += __shfl_xor(s, 2, 64);
    s += __shfl_xor(s, 4, 64);
    s += __shfl_xor(s, 8, 64);
    if ((lane & 15) == 0 && c < D) {
      const int hd = c / DH;
      const size_t i = ((size_t)b * a.H + hd) * a.N + j;
      a.delta[i] = s;
      // second half of the delta buffer: the log-sum-exp in log2 units, so
      // the backward kernels form exp2(s * scale * log2e - lse2) with one fma
      a.delta[(size_t)a.B * a.H * a.N + i] = a.lse[i] * LOG2E;
    }
  }
}

// ============================================================== dK, dV
constexpr int KV_KB = 128, KV_QT = 64;
constexpr int KV_S = DH + 8;       // [q][d] tiles
constexpr int KV_T = KV_QT + 8;    // [d][q] tiles

__global__ __launch_bounds__(256) void attn_bwd_kv_mfma_k(AttnBwd a) {
  __shared__ __attribute__((aligned(16))) uint16_t Qs[KV_QT * KV_S];
  __shared__ __attribute__((aligned(16))) uint16_t Gs[KV_QT * KV_S];
  __shared__ __attribute__((aligned(16))) uint16_t Qt[DH * KV_T];
  __shared__ __attribute__((aligned(16))) uint16_t Gt[DH * KV_T];
  __shared__ float Ls[KV_QT], Ds[KV_QT];
  const int bh = blockIdx.y, b = bh / a.H, hd = bh % a.H;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, h = lane >> 5, c32 = lane & 31;
  const int key = blockIdx.x * KV_KB + w * 32 + c32;
  const size_t base = (size_t)bh * a.N * DH;
  const uint16_t* Q = (const uint16_t*)a.Q + base;
  const uint16_t* K = (const uint16_t*)a.K + base;
  const uint16_t* V = (const uint16_t*)a.V + base;
  const uint16_t* G = (const uint16_t*)a.dO;
  const float sc = rsqrtf((float)DH);
  const int N = a.N;

  // threads [0, NB) stage Q blocks, [NB, 2 NB) dO blocks; lse and delta of
  // the tile are loaded by threads [0, KV_QT) and [KV_QT, 2 KV_QT)
  constexpr int NB = Tile8<KV_QT>::NBLK;
  constexpr int NT = KV_QT / 32;  // 32x32 score tiles per wave per query tile
  static_assert(2 * NB <= 256 && 2 * KV_QT <= 256, "tile too large for one block");
  Tile8<KV_QT> tq;
  const int tid = threadIdx.x;
  const bool isq = tid < NB;
  tq.init(tid < 2 * NB ? (isq ? tid : tid - NB) : -1);
  auto rows = [&](int i) -> const uint16_t* {
    if (i >= N) return nullptr;
    return isq ? Q + (size_t)i * DH : G + (size_t)row_of_tok_m(a.rm, b, i) * a.ld_do + hd * DH;
  };
  float lsv = 0.f;
  auto load_ld = [&](int q0) {
    if (tid < KV_QT) {
      const int qq = q0 + tid;
      lsv = qq < N ? a.lse[(size_t)bh * N + qq] : INFINITY;
    } else if (tid < 2 * KV_QT) {
      const int qq = q0 + tid - KV_QT;
      lsv = qq < N ? a.delta[(size_t)bh * N + qq] : 0.f;
    }
  };

  bf16x8 kf[8], vf[8];
#pragma unroll
  for (int kb = 0; kb < 8; ++kb) {
    if (key < N) {
      kf[kb] = ld8(K + (size_t)key * DH + kb * 16 + h * 8);
      vf[kb] = ld8(V + (size_t)key * DH + kb * 16 + h * 8);
    } else {
      kf[kb] = vf[kb] = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
    }
  }
  f32x16 dv[4], dk[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) { dv[i] = zero16(); dk[i] = zero16(); }

  tq.load(rows, 0);
  load_ld(0);
  for (int q0 = 0; q0 < N; q0 += KV_QT) {
    __syncthreads();
    if (isq) { tq.commit_rows<KV_S>(Qs); tq.commit_cols<KV_T>(Qt); }
    else { tq.commit_rows<KV_S>(Gs); tq.commit_cols<KV_T>(Gt); }
    if (tid < KV_QT) Ls[tid] = lsv;
    else if (tid < 2 * KV_QT) Ds[tid - KV_QT] = lsv;
    __syncthreads();
    if (q0 + KV_QT < N) { tq.load(rows, q0 + KV_QT); load_ld(q0 + KV_QT); }
    f32x16 s[NT], dp[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      s[t] = zero16();
      dp[t] = zero16();
#pragma unroll
      for (int kb = 0; kb < 8; ++kb) {
        s[t] = mfma(ld8(Qs + (32 * t + c32) * KV_S + kb * 16 + h * 8), kf[kb], s[t]);
        dp[t] = mfma(ld8(Gs + (32 * t + c32) * KV_S + kb * 16 + h * 8), vf[kb], dp[t]);
      }
    }
    // lane: key column, query rows 32t + 8(e/4) + 4h + e%4
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const float4 L4 = *(const float4*)(Ls + 32 * t + 8 * g + 4 * h);
        const float4 D4 = *(const float4*)(Ds + 32 * t + 8 * g + 4 * h);
        const float Lv[4] = {L4.x, L4.y, L4.z, L4.w}, Dv[4] = {D4.x, D4.y, D4.z, D4.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int e = 4 * g + i;
          const float p = __builtin_amdgcn_exp2f((s[t][e] * sc - Lv[i]) * LOG2E);
          s[t][e] = p;
          dp[t][e] = p * (dp[t][e] - Dv[i]);
        }
      }
#pragma unroll
    for (int c = 0; c < 2 * NT; ++c) {
      const bf16x8 pb = pack8(s[c >> 1], c & 1), db = pack8(dp[c >> 1], c & 1);
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        dv[dt] = mfma(ld4x2(Gt + (32 * dt + c32) * KV_T + 16 * c + 4 * h), pb, dv[dt]);
        dk[dt] = mfma(ld4x2(Qt + (32 * dt + c32) * KV_T + 16 * c + 4 * h), db, dk[dt]);
      }
    }
  }
  if (key >= N) return;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x4 vk, vv;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        vk[i] = (__bf16)(dk[dt][4 * g + i] * sc);
        vv[i] = (__bf16)dv[dt][4 * g + i];
      }
      const size_t off = base + (size_t)key * DH + 32 * dt + 8 * g + 4 * h;
      *(bf16x4*)((uint16_t*)a.dK + off) = vk;
      *(bf16x4*)((uint16_t*)a.dV + off) = vv;
    }
}

// ============================================================== dQ
constexpr int Q_QB = 128, Q_KT = 64;
constexpr int Q_S = DH + 8;
constexpr int Q_T = Q_KT + 8;

__global__ __launch_bounds__(256) void attn_bwd_q_mfma_k(AttnBwd a) {
  __shared__ __attribute__((aligned(16))) uint16_t Ks[Q_KT * Q_S];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[Q_KT * Q_S];
  __shared__ __attribute__((aligned(16))) uint16_t Kt[DH * Q_T];
  const int bh = blockIdx.y, b = bh / a.H;
  const int hd = bh % a.H;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, h = lane >> 5, c32 = lane & 31;
  const int q = blockIdx.x * Q_QB + w * 32 + c32;
  const size_t base = (size_t)bh * a.N * DH;
  const uint16_t* Q = (const uint16_t*)a.Q + base;
  const uint16_t* K = (const uint16_t*)a.K + base;
  const uint16_t* V = (const uint16_t*)a.V + base;
  const float sc = rsqrtf((float)DH);
  const int N = a.N;

  // threads [0, NB) stage K blocks (rows and columns), [NB, 2 NB) V blocks (rows)
  constexpr int NB = Tile8<Q_KT>::NBLK;
  constexpr int NT = Q_KT / 32;
  static_assert(2 * NB <= 256, "tile too large for one block");
  Tile8<Q_KT> tkv;
  const int tid = threadIdx.x;
  const bool isk = tid < NB;
  tkv.init(tid < 2 * NB ? (isk ? tid : tid - NB) : -1);
  const uint16_t* src = isk ? K : V;
  auto rows = [&](int i) -> const uint16_t* { return i < N ? src + (size_t)i * DH : nullptr; };

  bf16x8 qf[8], gf[8];
  const bool qv = q < N;
  const uint16_t* G = (const uint16_t*)a.dO + (qv ? (size_t)row_of_tok_m(a.rm, b, q) * a.ld_do + hd * DH : 0);
#pragma unroll
  for (int kb = 0; kb < 8; ++kb) {
    if (qv) {
      qf[kb] = ld8(Q + (size_t)q * DH + kb * 16 + h * 8);
      gf[kb] = ld8(G + kb * 16 + h * 8);
    } else {
      qf[kb] = gf[kb] = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
    }
  }
  const float L = qv ? a.lse[(size_t)bh * N + q] * LOG2E : INFINITY;
  const float Dl = qv ? a.delta[(size_t)bh * N + q] : 0.f;
  f32x16 dq[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) dq[i] = zero16();

  tkv.load(rows, 0);
  for (int k0 = 0; k0 < N; k0 += Q_KT) {
    __syncthreads();
    if (isk) { tkv.commit_rows<Q_S>(Ks); tkv.commit_cols<Q_T>(Kt); }
    else tkv.commit_rows<Q_S>(Vs);
    __syncthreads();
    if (k0 + Q_KT < N) tkv.load(rows, k0 + Q_KT);
    f32x16 s[NT], dp[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      s[t] = zero16();
      dp[t] = zero16();
#pragma unroll
      for (int kb = 0; kb < 8; ++kb) {
        s[t] = mfma(ld8(Ks + (32 * t + c32) * Q_S + kb * 16 + h * 8), qf[kb], s[t]);
        dp[t] = mfma(ld8(Vs + (32 * t + c32) * Q_S + kb * 16 + h * 8), gf[kb], dp[t]);
      }
    }
    // lane: query column, key rows 32t + 8(e/4) + 4h + e%4
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int kk = k0 + 32 * t + 8 * (e >> 2) + 4 * h + (e & 3);
        const float p = kk < N ? __builtin_amdgcn_exp2f(s[t][e] * sc * LOG2E - L) : 0.f;
        dp[t][e] = p * (dp[t][e] - Dl);
      }
#pragma unroll
    for (int c = 0; c < 2 * NT; ++c) {
      const bf16x8 db = pack8(dp[c >> 1], c & 1);
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) dq[dt] = mfma(ld4x2(Kt + (32 * dt + c32) * Q_T + 16 * c + 4 * h), db, dq[dt]);
    }
  }
  if (!qv) return;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x4 v;
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = (__bf16)(dq[dt][4 * g + i] * sc);
      *(bf16x4*)((uint16_t*)a.dQ + base + (size_t)q * DH + 32 * dt + 8 * g + 4 * h) = v;
    }
}

// ====================================================== backward, v2
// Tiles of 64 rows x 128 (one head) are fetched straight into LDS by buffer
// loads with the LDS bit (no register staging), three k tiles in flight, one
// barrier per tile.  A tile is stored unpadded, 256 B per row, with the 16-byte
// chunks of row r XOR-swizzled by asw(r); the table makes both fragment
// patterns conflict-free whether the LDS serves 8 or 16 lanes per cycle:
//   row fragments (16-byte reads, 8/16 consecutive rows, one chunk) and
//   transposed fragments (ds_read_b64_tr_b16: 4 consecutive rows x 32 B per
//   16 lanes), which replace the transposed tile copies: lane i of a 16-lane
//   group receives element (row e, column i) of the 4 x 16 block the group
//   fetched, so two such reads give the A operand of a product that contracts
//   over the tile rows, in the row order the accumulator-fed B operand uses.
constexpr unsigned long long ASW = 0xf953e842db71ca60ull;
__device__ __forceinline__ int asw(int r) { return (int)((ASW >> (4 * (r & 15))) & 15); }
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
#define ALDS(p) ((__attribute__((address_space(3))) void*)(p))
// byte address of a shared-memory location in the LDS aperture
__device__ inline unsigned lds_addr(const void* p) {
  return (unsigned)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}
constexpr int AOOB = 0x7ffffff0;  // buffer offset past any resource: loads return zero

__device__ __forceinline__ __amdgpu_buffer_rsrc_t arsrc(const void* p, long bytes) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)p, (short)0, (int)bytes, 0x00020000);
}

// Per-lane constants of one 64-row tile: direct-load slots and fragment offsets.
struct ATile {
  int lrow[4], lchunk[4];  // direct loads: tile row and source chunk of this lane, per load
  int roff[8];             // row fragment, k16 step kb: byte offset for tile row (lane % 32)
  int t1[4], t2[4];        // transposed fragment, 32-column block dt: the two reads
  __device__ inline void init() {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      lrow[t] = 4 * (wave * 4 + t) + lane / 16;
      lchunk[t] = (lane % 16) ^ asw(lrow[t]);
    }
    const int rr = lane & 31, h = lane >> 5;
#pragma unroll
    for (int kb = 0; kb < 8; ++kb) roff[kb] = rr * 256 + (((2 * kb + h) ^ asw(rr)) << 4);
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const int2 o = tr_off(lane, dt);
      t1[dt] = o.x;
      t2[dt] = o.y;
    }
  }
  // byte offsets of the two transposing reads of column block dt for this lane
  static __device__ inline int2 tr_off(int lane, int dt) {
    const int g = lane >> 4, j = lane & 15;
    const int q1 = 4 * (g >> 1) + (j >> 2), q2 = q1 + 8;
    const int ch = 4 * dt + 2 * (g & 1) + ((j & 3) >> 1);
    return {q1 * 256 + ((ch ^ asw(q1)) << 4) + (j & 1) * 8, q2 * 256 + ((ch ^ asw(q2)) << 4) + (j & 1) * 8};
  }
  // 16 direct loads of 1 KB (4 rows each), 4 per wave; rowoff(r) = byte offset
  // of tile row r in the resource, or a negative value for a padding row
  template <class RowOff>
  __device__ inline void load(__amdgpu_buffer_rsrc_t R, char* S, RowOff rowoff) const {
    // wave-uniform: the LDS destination (M0) is then computed on the scalar unit
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int ro = rowoff(lrow[t]);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(R, ALDS(S + (wave * 4 + t) * 1024), 16, ro < 0 ? AOOB : ro + lchunk[t] * 16,
                                               0, 0, 0);
    }
  }
  // the same 16 loads with precomputed byte offsets off[t] (AOOB: a padding row)
  __device__ inline void load_at(__amdgpu_buffer_rsrc_t R, char* S, const int* off) const {
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
    for (int t = 0; t < 4; ++t)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(R, ALDS(S + (wave * 4 + t) * 1024), 16, off[t], 0, 0, 0);
  }
  // A fragment of rows 32t + (lane % 32), elements 16kb + 8(lane / 32) .. +7
  __device__ inline bf16x8 row(const char* S, int t, int kb) const {
    return __builtin_bit_cast(bf16x8, *(const u32x4*)(S + roff[kb] + t * 8192));
  }
  // A fragment of the transposed tile: row d = 32dt + (lane % 32), contraction
  // slots = tile rows 16c + 4(lane / 32) + 0..3 and 16c + 8 + 4(lane / 32) + 0..3
  __device__ inline bf16x8 tr(const char* S, int c, int dt) const {
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(S + t1[dt] + c * 4096));
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(S + t2[dt] + c * 4096));
    const s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
  }
  // The two read offsets of column block dt, for a dt known only at run time:
  // recomputed rather than indexed, so that t1/t2 stay in registers (a dynamic
  // index moves the arrays to LDS and costs a strided LDS read per use)
  __device__ inline int2 tr_sel(int dt) const { return tr_off(threadIdx.x & 63, dt); }
  __device__ inline bf16x8 tr(const char* S, int c, int2 o) const {
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(S + o.x + c * 4096));
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(S + o.y + c * 4096));
    const s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
  }
};

// LDS barrier for the direct-loaded stages: this wave's loads older than its
// newest NL are done (they are LDS writes), its LDS reads are done, then
// s_barrier.  No release fence: __syncthreads would wait for every direct
// load still in flight.  The empty asm statements keep the compiler from
// moving memory accesses across it.
template <int NL>
__device__ __forceinline__ void attn_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((NL & 15) | ((NL >> 4) << 14) | 0x70);  // vmcnt(NL) expcnt(7) lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Fragment reads of the direct-loaded tiles with two registers of per-lane
// offsets: the row fragment of k16 step kb is at roff0 ^ (kb << 5) and the
// transposing reads of column block dt at t10 ^ (dt << 6), t20 ^ (dt << 6)
// (the swizzle XORs the 16-byte chunk index, and kb and dt select its upper
// bits), so one offset per pattern serves all steps.
struct ATileX {
  int roff0, t10, t20;
  __device__ inline void init() {
    const int lane = threadIdx.x & 63, rr = lane & 31, h = lane >> 5;
    roff0 = rr * 256 + ((h ^ asw(rr)) << 4);
    const int2 o = ATile::tr_off(lane, 0);
    t10 = o.x;
    t20 = o.y;
  }
  __device__ inline bf16x8 row(const char* S, int t, int kb) const {
    return __builtin_bit_cast(bf16x8, *(const u32x4*)(S + (roff0 ^ (kb << 5)) + t * 8192));
  }
  __device__ inline bf16x8 tr(const char* S, int c, int dt) const {
    const s16x4 lo =
        __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(S + (t10 ^ (dt << 6)) + c * 4096));
    const s16x4 hi =
        __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(S + (t20 ^ (dt << 6)) + c * 4096));
    const s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
  }
};

// ------------------------------------------------------------ dK, dV (v5)
// Two waves per SIMD: eight waves per workgroup of 128 keys.  Wave w takes
// the 32 keys 32 (w % 4) .. of the block and the 32-query half w / 4 of every
// 64-query tile.  K and V of the block stay in LDS and are read as B
// fragments, so that a wave fits in 256 registers; the two waves of a key
// group add their partial dV and dK through LDS at the end, in fixed order.
// Query tiles stream through two stages, one barrier per tile.  No mask: rows
// of Q, dO, log-sum-exp and delta past N load as zeros, which gives a padded
// query dP = 0 and delta = 0, hence dS = 0 and no share of dV or dK; the tile
// count is rounded up to the two-stage unroll with zero tiles, and dS^T stores
// past the padded width fall outside the store resource.
constexpr int KV5_KB = 128, KV5_QT = 64;

template <bool DS>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_bwd_kv5_k(AttnBwd a) {
  // K | V of the block, and per stage Q | dO of a query tile: the second
  // operand of each array sits at a fixed offset from the first, so one
  // offset register per read pattern serves both
  __shared__ __attribute__((aligned(1024))) char KV[65536], QG0[32768], QG1[32768];
  __shared__ __attribute__((aligned(256))) float L0[64], D0[64], L1[64], D1[64];
  const int bh = blockIdx.y, b = bh / a.H, hd = bh % a.H;
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), h = lane >> 5, c32 = lane & 31;
  const int kg = w & 3, th = w >> 2;  // key group, query half
  const int key = blockIdx.x * KV5_KB + kg * 32 + c32;
  const int N = a.N;
  const size_t base = (size_t)bh * N * DH;
  const float sc = rsqrtf((float)DH), scl = sc * LOG2E;
  const __amdgpu_buffer_rsrc_t RK = arsrc((const uint16_t*)a.K + base, (long)N * DH * 2);
  const __amdgpu_buffer_rsrc_t RV = arsrc((const uint16_t*)a.V + base, (long)N * DH * 2);
  const __amdgpu_buffer_rsrc_t RQ = arsrc((const uint16_t*)a.Q + base, (long)N * DH * 2);
  const __amdgpu_buffer_rsrc_t RG = arsrc(a.dO, (long)a.rm.rows() * a.ld_do * 2);
  const __amdgpu_buffer_rsrc_t RL = arsrc(a.delta + (size_t)a.B * a.H * N + (size_t)bh * N, (long)N * 4);
  const __amdgpu_buffer_rsrc_t RD = arsrc(a.delta + (size_t)bh * N, (long)N * 4);
  // this head's dS^T chunks; this lane's key row in its key block
  const __amdgpu_buffer_rsrc_t RS =
      arsrc(DS ? (const uint16_t*)a.dS + (size_t)bh * a.nk_pad * a.ld_ds : nullptr, DS ? (long)a.nk_pad * a.ld_ds * 2 : 0);
  const int srow = (blockIdx.x * KV5_KB * a.ld_ds + (kg * 32 + c32) * 64) * 2;
  ATileX at;  // fragment offsets (the direct-load slots below are for 8 waves)
  at.init();

  // direct loads for 8 waves: 1 KB slot s holds rows 4s .. 4s+3
  auto slot_off = [&](int s) {
    const int row = 4 * s + lane / 16;
    return int2{row, ((lane % 16) ^ asw(row)) << 4};
  };
  // K and V of the block: 32 slots each, 4 per wave
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int s = 4 * w + t;
    const int2 o = slot_off(s);
    const int off = (blockIdx.x * KV5_KB + o.x) * (DH * 2) + o.y;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(RK, ALDS(KV + s * 1024), 16, off, 0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(RV, ALDS(KV + 32768 + s * 1024), 16, off, 0, 0, 0);
  }
  // query tiles: 16 slots per operand, 2 per wave
  const int gofs_t = b * a.rm.nt, gofs_i = a.rm.B * a.rm.nt + b * a.rm.ni - a.rm.nt;
  const int grow = a.ld_do * 2, nt = a.rm.nt;
  auto load_tile = [&](char* Qd, float* Ld, float* Dd, int q0) {
    char* const Gd = Qd + 16384;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int2 o = slot_off(2 * w + t);
      const int q = q0 + o.x;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(RQ, ALDS(Qd + (2 * w + t) * 1024), 16, q * (DH * 2) + o.y, 0, 0, 0);
      const int og = q < N ? __mul24(q + (q < nt ? gofs_t : gofs_i), grow) + hd * DH * 2 + o.y : AOOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(RG, ALDS(Gd + (2 * w + t) * 1024), 16, og, 0, 0, 0);
    }
    if (w == 0) __builtin_amdgcn_raw_ptr_buffer_load_lds(RL, ALDS(Ld), 4, (q0 + lane) * 4, 0, 0, 0);
    if (w == 1) __builtin_amdgcn_raw_ptr_buffer_load_lds(RD, ALDS(Dd), 4, (q0 + lane) * 4, 0, 0, 0);
  };

  f32x16 dv[4], dk[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) { dv[i] = zero16(); dk[i] = zero16(); }
  const int ntile = ((N + KV5_QT - 1) / KV5_QT + 1) & ~1;
  load_tile(QG0, L0, D0, 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  // V is used only for dP; negated once in LDS, the dP products accumulate
  // onto delta and give delta - dP, so that dS = -P (delta - dP) needs no
  // subtraction per element (padding rows: delta = 0, dO = 0, so still 0)
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    u32x4* vp = (u32x4*)(KV + 32768) + i * 512 + threadIdx.x;
    u32x4 x = *vp;
    x ^= 0x80008000u;
    *vp = x;
  }
  __syncthreads();

  auto iter = [&](auto ic, int it) {
    constexpr int c = decltype(ic)::value;
    char* Qc = c == 0 ? QG0 : QG1;
    const float* Lc = c == 0 ? L0 : L1;
    const float* Dc = c == 0 ? D0 : D1;
    const int q0 = it * KV5_QT;
    // tile it has landed (only the previous tile's 2 dS^T stores may fly); the
    // other stage was last read in the previous iteration
    attn_barrier<DS ? 2 : 0>();
    if constexpr (c == 0) load_tile(QG1, L1, D1, q0 + KV5_QT);
    else load_tile(QG0, L0, D0, q0 + KV5_QT);
    // per-iteration opaque copies of the offsets, as LDS addresses (the
    // array's base included, so that a read needs no add: the base is a
    // multiple of 1024 and the XORed bits lie below it); the address
    // arithmetic is redone in each iteration instead of kept in registers
    // across the loop
    const unsigned bq = lds_addr(Qc), bk = lds_addr(KV);
    unsigned qo = at.roff0 + th * 8192 + bq, ko = at.roff0 + kg * 8192 + bk;
    unsigned t1 = at.t10 + th * 8192 + bq, t2 = at.t20 + th * 8192 + bq;
    asm volatile("" : "+v"(qo), "+v"(ko), "+v"(t1), "+v"(t2));
    // row fragment of k16 step kb at byte cofs of array S (base b)
    auto rowf = [&](const char* S, unsigned b, unsigned o, int kb, int cofs) {
      return __builtin_bit_cast(bf16x8, *(const u32x4*)(S + ((o ^ (kb << 5)) - b) + cofs));
    };
    auto trf = [&](int blk, int dt, int cofs) {
      const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) s16x4*)(Qc + ((t1 ^ (dt << 6)) - bq) + blk * 4096 + cofs));
      const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) s16x4*)(Qc + ((t2 ^ (dt << 6)) - bq) + blk * 4096 + cofs));
      const s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      return __builtin_bit_cast(bf16x8, v);
    };
    // S and dP of this wave's keys and query half (lane: key column, query
    // rows 32 th + 8(e/4) + 4h + e%4)
    f32x16 st = zero16(), dpt;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const float4 D4 = *(const float4*)(Dc + 32 * th + 8 * g + 4 * h);
      dpt[4 * g] = D4.x;
      dpt[4 * g + 1] = D4.y;
      dpt[4 * g + 2] = D4.z;
      dpt[4 * g + 3] = D4.w;
    }
#pragma unroll
    for (int kb = 0; kb < 8; ++kb) {
      st = mfma(rowf(Qc, bq, qo, kb, 0), rowf(KV, bk, ko, kb, 0), st);
      dpt = mfma(rowf(Qc, bq, qo, kb, 16384), rowf(KV, bk, ko, kb, 32768), dpt);
    }
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const float4 L4 = *(const float4*)(Lc + 32 * th + 8 * g + 4 * h);
      const float Lv[4] = {L4.x, L4.y, L4.z, L4.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int e = 4 * g + i;
        const float p = __builtin_amdgcn_exp2f(fmaf(st[e], scl, -Lv[i]));
        st[e] = p;
        dpt[e] = -p * dpt[e];
      }
    }
    // dS^T of the half's 16-query block blk: lane (c32, h) holds queries
    // 4h + 0..3 and 8 + 4h + 0..3; swapping the upper half-wave's first pair of
    // dwords with the lower half-wave's second pair leaves it queries
    // 8h + 0..7, one 16-byte store.  Columns past the padded width fall
    // outside the resource.
    const unsigned so = q0 < a.ld_ds ? (unsigned)(srow + q0 * KV5_KB * 2 + 64 * th + 16 * h) : (unsigned)AOOB;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      const bf16x8 pb = pack8(st, blk), db = pack8(dpt, blk);
      if constexpr (DS) {
        const u32x4 u = __builtin_bit_cast(u32x4, db);
        const auto s0 = __builtin_amdgcn_permlane32_swap(u[0], u[2], false, false);
        const auto s1 = __builtin_amdgcn_permlane32_swap(u[1], u[3], false, false);
        __builtin_amdgcn_raw_buffer_store_b128(u32x4{s0[0], s1[0], s0[1], s1[1]}, RS, (int)(so + 32 * blk), 0, 0);
      }
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        dv[dt] = mfma(trf(blk, dt, 16384), pb, dv[dt]);
        dk[dt] = mfma(trf(blk, dt, 0), db, dk[dt]);
      }
    }
  };
  for (int it = 0; it < ntile; it += 2) {
    iter(std::integral_constant<int, 0>(), it);
    iter(std::integral_constant<int, 1>(), it + 1);
  }
  // the two query halves of a key group: waves 4..7 hand their partial sums
  // to waves 0..3 through LDS (dV, then dK), which add them in that order
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  float* const xs = (float*)KV + kg * 4096;  // 16 KB per key group
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    f32x16* acc = pass == 0 ? dv : dk;
    if (th == 1) {
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int g = 0; g < 4; ++g)
          *(float4*)(xs + ((dt * 4 + g) * 64 + lane) * 4) =
              make_float4(acc[dt][4 * g], acc[dt][4 * g + 1], acc[dt][4 * g + 2], acc[dt][4 * g + 3]);
    }
    __syncthreads();
    if (th == 0) {
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const float4 o = *(const float4*)(xs + ((dt * 4 + g) * 64 + lane) * 4);
          acc[dt][4 * g] += o.x;
          acc[dt][4 * g + 1] += o.y;
          acc[dt][4 * g + 2] += o.z;
          acc[dt][4 * g + 3] += o.w;
        }
    }
    __syncthreads();
  }
  if (th != 0 || key >= N) return;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x4 vk, vv;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        vk[i] = (__bf16)(dk[dt][4 * g + i] * sc);
        vv[i] = (__bf16)dv[dt][4 * g + i];
      }
      const size_t off = base + (size_t)key * DH + 32 * dt + 8 * g + 4 * h;
      *(bf16x4*)((uint16_t*)a.dK + off) = vk;
      *(bf16x4*)((uint16_t*)a.dV + off) = vv;
    }
}

// ------------------------------------------------------------ forward (v2)
// 128 queries per workgroup (32 per wave, Q^T fragments in registers); key
// tiles of 64 rows of K and V stream through two LDS stages by direct loads,
// one barrier per tile.  Two stages (64 KB) and 246 registers let two
// workgroups share a CU, so that one's softmax work overlaps the other's
// MFMAs (with three stages and one workgroup per CU the kernel was 1.3x
// slower).  S^T = K Q^T from row fragments of the K tile;
// O^T += V^T P^T from transposing reads of the V tile, in the contraction-slot
// order of the accumulator-fed P^T.  Rows of K and V past N load as zeros; the
// keys past N are masked in the ragged last tile only.
constexpr int F2_QB = 128, F2_KT = 64;
constexpr float F2_SLACK = 8.f;

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_fwd2_k(AttnFwd a) {
  __shared__ __attribute__((aligned(1024))) char K0[16384], V0[16384], K1[16384], V1[16384];
  const int bh = blockIdx.y, b = bh / a.H, hd = bh % a.H;
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), h = lane >> 5, c32 = lane & 31;
  const int q = blockIdx.x * F2_QB + w * 32 + c32;  // this lane's query
  const int N = a.N;
  const size_t base = (size_t)bh * N * DH;
  const uint16_t* Q = (const uint16_t*)a.Q + base;
  const float sc = rsqrtf((float)DH) * LOG2E;
  const __amdgpu_buffer_rsrc_t RK = arsrc((const uint16_t*)a.K + base, (long)N * DH * 2);
  const __amdgpu_buffer_rsrc_t RV = arsrc((const uint16_t*)a.V + base, (long)N * DH * 2);
  ATile at;
  at.init();
  // per load slot: byte offset of the lane's chunk in a tile at k0 = 0
  int koff[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) koff[t] = at.lrow[t] * (DH * 2) + at.lchunk[t] * 16;
  auto load_tile = [&](char* Kd, char* Vd, int k0) {
    int o[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) o[t] = koff[t] + k0 * (DH * 2);
    at.load_at(RK, Kd, o);
    at.load_at(RV, Vd, o);
  };

  bf16x8 qf[8];
#pragma unroll
  for (int kb = 0; kb < 8; ++kb) {
    if (q < N) qf[kb] = ld8(Q + (size_t)q * DH + kb * 16 + h * 8);
    else qf[kb] = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
  }
  f32x16 o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = zero16();
  float m = -INFINITY, l = 0.f;

  const int ntile = (N + F2_KT - 1) / F2_KT, nfull = N / F2_KT;
  load_tile(K0, V0, 0);
  // one key tile; MASK: the ragged last tile (no further loads)
  auto iter = [&](auto ic, auto mc, int it) {
    constexpr int c = decltype(ic)::value;
    constexpr bool MASK = decltype(mc)::value;
    const char* Kc = c == 0 ? K0 : K1;
    const char* Vc = c == 0 ? V0 : V1;
    const int k0 = it * F2_KT;
    // tile it has landed (its loads are this wave's last); the other stage,
    // for tile it+1, was last read in the previous iteration
    attn_barrier<0>();
    if constexpr (!MASK) {
      if constexpr (c == 0) load_tile(K1, V1, k0 + F2_KT);
      else load_tile(K0, V0, k0 + F2_KT);
    }
    // S^T: lane = query column, key rows 32t + 8(e/4) + 4h + e%4
    f32x16 st[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      bf16x8 fk[8];
#pragma unroll
      for (int kb = 0; kb < 8; ++kb) fk[kb] = at.row(Kc, t, kb);
      st[t] = mfma(fk[0], qf[0], zero16());
#pragma unroll
      for (int kb = 1; kb < 8; ++kb) st[t] = mfma(fk[kb], qf[kb], st[t]);
    }
    // row maximum of the raw scores (the scale is positive)
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        if (MASK && k0 + 32 * t + 8 * (e >> 2) + 4 * h + (e & 3) >= N) st[t][e] = -INFINITY;
        mx = fmaxf(mx, st[t][e]);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * sc;
    // The reference point m moves only when a row's maximum passes it by more
    // than F2_SLACK (log2 units): P = 2^(s - m) then stays below 2^F2_SLACK,
    // and the rescale of O and l is skipped on the tiles where no row of the
    // wave moves (after the first tiles, nearly all of them).
    if (__builtin_amdgcn_ballot_w64(mx > m + F2_SLACK)) {
      const float mn = fmaxf(m, mx);
      const float corr = __builtin_amdgcn_exp2f(m - mn);
      l *= corr;
      m = mn;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[i][e] *= corr;
    }
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float p = __builtin_amdgcn_exp2f(fmaf(st[t][e], sc, -m));
        st[t][e] = p;
        l += p;
      }
    // O^T += V^T P^T, 16 keys (tile rows 16 cb ..) per step
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      const bf16x8 pb = pack8(st[cb >> 1], cb & 1);
      bf16x8 tv[4];
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) tv[dt] = at.tr(Vc, cb, dt);
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) o[dt] = mfma(tv[dt], pb, o[dt]);
    }
  };
  using F = std::false_type;
  using T = std::true_type;
  int it = 0;
  for (; it + 1 < nfull; it += 2) {
    iter(std::integral_constant<int, 0>(), F(), it);
    iter(std::integral_constant<int, 1>(), F(), it + 1);
  }
  if (it < nfull) iter(std::integral_constant<int, 0>(), F(), it);
  if (nfull < ntile) {  // ragged last tile
    if (nfull % 2 == 0) iter(std::integral_constant<int, 0>(), T(), nfull);
    else iter(std::integral_constant<int, 1>(), T(), nfull);
  }
  // no direct load may still be landing when the workgroup's LDS is released
  __builtin_amdgcn_s_waitcnt(0);
  l += __shfl_xor(l, 32, 64);
  if (q >= N) return;
  const float inv = 1.f / l;
  uint16_t* O = (uint16_t*)a.O + (size_t)row_of_tok_m(a.rm, b, q) * a.ld_o + hd * DH;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x4 v;
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = (__bf16)(o[dt][4 * g + i] * inv);
      *(bf16x4*)(O + 32 * dt + 8 * g + 4 * h) = v;
    }
  if (h == 0) a.lse[(size_t)bh * N + q] = (m + __log2f(l)) * LN2;
}

// ------------------------------------------------------------ dQ (v2)
// 128 queries per workgroup (32 per wave, Q and dO fragments in registers);
// key tiles of 64 rows of K and V stream through three LDS stages.
constexpr int Q2_QB = 128, Q2_KT = 64;

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void attn_bwd_q2_k(AttnBwd a) {
  __shared__ __attribute__((aligned(1024))) char K0[16384], V0[16384], K1[16384], V1[16384], K2[16384], V2[16384];
  const int bh = blockIdx.y, b = bh / a.H, hd = bh % a.H;
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), h = lane >> 5, c32 = lane & 31;
  const int q = blockIdx.x * Q2_QB + w * 32 + c32;
  const int N = a.N;
  const size_t base = (size_t)bh * N * DH;
  const uint16_t* Q = (const uint16_t*)a.Q + base;
  const float sc = rsqrtf((float)DH), scl = sc * LOG2E;
  const __amdgpu_buffer_rsrc_t RK = arsrc((const uint16_t*)a.K + base, (long)N * DH * 2);
  const __amdgpu_buffer_rsrc_t RV = arsrc((const uint16_t*)a.V + base, (long)N * DH * 2);
  ATile at;
  at.init();

  bf16x8 qf[8], gf[8];
  const bool qv = q < N;
  const uint16_t* G = (const uint16_t*)a.dO + (qv ? (size_t)row_of_tok_m(a.rm, b, q) * a.ld_do + hd * DH : 0);
#pragma unroll
  for (int kb = 0; kb < 8; ++kb) {
    if (qv) {
      qf[kb] = ld8(Q + (size_t)q * DH + kb * 16 + h * 8);
      gf[kb] = ld8(G + kb * 16 + h * 8);
    } else {
      qf[kb] = gf[kb] = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
    }
  }
  const float L = qv ? a.lse[(size_t)bh * N + q] * LOG2E : INFINITY;
  const float Dl = qv ? a.delta[(size_t)bh * N + q] : 0.f;
  f32x16 dq[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) dq[i] = zero16();

  auto load_tile = [&](char* Kd, char* Vd, int k0) {
    at.load(RK, Kd, [&](int r) { return (k0 + r) * (DH * 2); });
    at.load(RV, Vd, [&](int r) { return (k0 + r) * (DH * 2); });
  };
  const int ntile = (N + Q2_KT - 1) / Q2_KT;
  load_tile(K0, V0, 0);
  load_tile(K1, V1, Q2_KT);

  auto iter = [&](auto ic, auto mc, int it) {
    constexpr int c = decltype(ic)::value;
    constexpr bool MASK = decltype(mc)::value;
    char* Kc = c == 0 ? K0 : (c == 1 ? K1 : K2);
    char* Vc = c == 0 ? V0 : (c == 1 ? V1 : V2);
    const int k0 = it * Q2_KT;
    attn_barrier<8>();
    if constexpr (!MASK) {
      if constexpr (c == 0) load_tile(K2, V2, k0 + 2 * Q2_KT);
      else if constexpr (c == 1) load_tile(K0, V0, k0 + 2 * Q2_KT);
      else load_tile(K1, V1, k0 + 2 * Q2_KT);
    }
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      bf16x8 fk[8], fv[8];
#pragma unroll
      for (int kb = 0; kb < 8; ++kb) {
        fk[kb] = at.row(Kc, t, kb);
        fv[kb] = at.row(Vc, t, kb);
      }
      __builtin_amdgcn_sched_barrier(0);
      f32x16 st = mfma(fk[0], qf[0], zero16());
      f32x16 dpt = mfma(fv[0], gf[0], zero16());
#pragma unroll
      for (int kb = 1; kb < 8; ++kb) {
        st = mfma(fk[kb], qf[kb], st);
        dpt = mfma(fv[kb], gf[kb], dpt);
      }
      __builtin_amdgcn_sched_barrier(0);
      // lane: query column, key rows 32t + 8(e/4) + 4h + e%4
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        float p = __builtin_amdgcn_exp2f(fmaf(st[e], scl, -L));
        if (MASK && k0 + 32 * t + 8 * (e >> 2) + 4 * h + (e & 3) >= N) p = 0.f;
        dpt[e] = p * (dpt[e] - Dl);
      }
      __builtin_amdgcn_sched_barrier(0);
      bf16x8 tk[2][4];
#pragma unroll
      for (int half = 0; half < 2; ++half)
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) tk[half][dt] = at.tr(Kc, 2 * t + half, dt);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const bf16x8 db = pack8(dpt, half);
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) dq[dt] = mfma(tk[half][dt], db, dq[dt]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  using F = std::false_type;
  using T = std::true_type;
  const int nfull = N / Q2_KT;
  int it = 0;
  for (; it + 2 < nfull; it += 3) {
    iter(std::integral_constant<int, 0>(), F(), it);
    iter(std::integral_constant<int, 1>(), F(), it + 1);
    iter(std::integral_constant<int, 2>(), F(), it + 2);
  }
  if (it < nfull) iter(std::integral_constant<int, 0>(), F(), it);
  if (it + 1 < nfull) iter(std::integral_constant<int, 1>(), F(), it + 1);
  if (nfull < ntile) {
    switch (nfull % 3) {
      case 0: iter(std::integral_constant<int, 0>(), T(), nfull); break;
      case 1: iter(std::integral_constant<int, 1>(), T(), nfull); break;
      default: iter(std::integral_constant<int, 2>(), T(), nfull); break;
    }
  }
  __builtin_amdgcn_s_waitcnt(0);
  if (!qv) return;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x4 v;
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = (__bf16)(dq[dt][4 * g + i] * sc);
      *(bf16x4*)((uint16_t*)a.dQ + base + (size_t)q * DH + 32 * dt + 8 * g + 4 * h) = v;
    }
}

// ------------------------------------------------------------ dQ from dS^T
// dQ = dS K with dS^T as stored by the dK/dV kernel: 128 queries per
// workgroup, 64-key tiles of K and of dS^T stream through four LDS stages
// (three tiles in flight).  Per 16-key block c: the K^T fragments of the
// wave's 32-row head-dimension blocks and its dS^T fragment are transposing
// LDS reads in the same contraction-slot order; dQ^T += K^T dS^T.  No scores
// are recomputed: the pass is bound by reading dS^T once.  Eight waves, two
// per SIMD: wave w takes query block w % 4 (32 queries) and head-dimension
// half w / 4 (two 32-row blocks of dQ^T), so a wave that waits to issue its
// direct loads leaves the SIMD to the other wave's fragment reads and MFMAs.
// Each wave issues two of the sixteen 1 KB loads of each 64 x 128 tile.
constexpr int Q4_QB = 128, Q4_KT = 64;

__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_bwd_q4_k(AttnBwd a) {
  __shared__ __attribute__((aligned(1024))) char K0[16384], S0[16384], K1[16384], S1[16384], K2[16384], S2[16384],
      K3[16384], S3[16384];
  const int bh = blockIdx.y;
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), h = lane >> 5, c32 = lane & 31;
  const int qw = w & 3, dh = w >> 2;
  const int qb = blockIdx.x * Q4_QB;
  const int q = qb + qw * 32 + c32;
  const int N = a.N;
  const size_t base = (size_t)bh * N * DH;
  const float sc = rsqrtf((float)DH);
  const __amdgpu_buffer_rsrc_t RK = arsrc((const uint16_t*)a.K + base, (long)N * DH * 2);
  const __amdgpu_buffer_rsrc_t RS =
      arsrc((const uint16_t*)a.dS + (size_t)bh * a.nk_pad * a.ld_ds, (long)a.nk_pad * a.ld_ds * 2);
  ATile at;
  at.init();
  // direct-load slots of this wave: tile rows 4 (2w + t) + lane / 16, t = 0, 1;
  // sof[t]: the slot's byte offset in a tile of the chunked dS^T (a tile row
  // is 128 queries: source chunks 0-7 in the chunk of the block's first 64
  // queries, 8-15 in the next chunk, 16 KB on)
  // kof[t]: the slot's byte offset in a K tile at k0 = 0
  int sof[2], kof[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int lrow = 4 * (2 * w + t) + lane / 16, lch = (lane % 16) ^ asw(lrow);
    sof[t] = lrow * 128 + (lch >> 3) * 16384 + (lch & 7) * 16;
    kof[t] = lrow * (DH * 2) + lch * 16;
  }
  const int nqt = a.ld_ds / 64;
  const int2 wsel = at.tr_sel(qw), dsel0 = at.tr_sel(2 * dh), dsel1 = at.tr_sel(2 * dh + 1);
  f32x16 dq[2] = {zero16(), zero16()};
  auto load_tile = [&](char* Kd, char* Sd, int k0) {
    // K rows at or past N and key blocks past the padded count lie past
    // their resources and read as zeros; keys k0 .. k0+63 lie in key block
    // k0 / 128 of dS^T, rows (k0 % 128) ..
    const int kpart = k0 * (DH * 2), spart = ((k0 >> 7) * nqt + qb / 64) * 16384 + (k0 & 64) * 128;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
    for (int t = 0; t < 2; ++t)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(RK, ALDS(Kd + (2 * wave + t) * 1024), 16, kpart + kof[t], 0, 0, 0);
#pragma unroll
    for (int t = 0; t < 2; ++t)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(RS, ALDS(Sd + (2 * wave + t) * 1024), 16, spart + sof[t], 0, 0, 0);
  };
  // Every tile load is issued whether the tile exists or not, so that the
  // issue order (and the waits the compiler derives from it) is the same in
  // every iteration: K rows at or past N and dS^T rows past the padded key
  // count read as zeros through the resources' range checks.  The tile count
  // is rounded up to a multiple of 4; the extra tiles add exact zeros.
  const int ntile = ((N + Q4_KT - 1) / Q4_KT + 3) & ~3;
  load_tile(K0, S0, 0);
  load_tile(K1, S1, Q4_KT);
  load_tile(K2, S2, 2 * Q4_KT);
  auto iter = [&](auto ic, int it) {
    constexpr int c = decltype(ic)::value;
    char* Kc = c == 0 ? K0 : (c == 1 ? K1 : (c == 2 ? K2 : K3));
    char* Sc = c == 0 ? S0 : (c == 1 ? S1 : (c == 2 ? S2 : S3));
    const int k0 = it * Q4_KT;
    // tile it has landed once at most the loads of the two later tiles in
    // flight (4 direct loads per tile and wave) are outstanding
    attn_barrier<8>();
    // the stage of tile it+3 was last read in iteration it-1
    if constexpr (c == 0) load_tile(K3, S3, k0 + 3 * Q4_KT);
    else if constexpr (c == 1) load_tile(K0, S0, k0 + 3 * Q4_KT);
    else if constexpr (c == 2) load_tile(K1, S1, k0 + 3 * Q4_KT);
    else load_tile(K2, S2, k0 + 3 * Q4_KT);
    bf16x8 tk[2][2], ts[2];
    tk[0][0] = at.tr(Kc, 0, dsel0);
    tk[0][1] = at.tr(Kc, 0, dsel1);
    ts[0] = at.tr(Sc, 0, wsel);
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      const int cur = cb & 1, nxt = cur ^ 1;
      if (cb + 1 < 4) {
        tk[nxt][0] = at.tr(Kc, cb + 1, dsel0);
        tk[nxt][1] = at.tr(Kc, cb + 1, dsel1);
        ts[nxt] = at.tr(Sc, cb + 1, wsel);
      }
      dq[0] = mfma(tk[cur][0], ts[cur], dq[0]);
      dq[1] = mfma(tk[cur][1], ts[cur], dq[1]);
    }
  };
  for (int it = 0; it < ntile; it += 4) {
    iter(std::integral_constant<int, 0>(), it);
    iter(std::integral_constant<int, 1>(), it + 1);
    iter(std::integral_constant<int, 2>(), it + 2);
    iter(std::integral_constant<int, 3>(), it + 3);
  }
  __builtin_amdgcn_s_waitcnt(0);
  if (q >= N) return;
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x4 v;
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = (__bf16)(dq[j][4 * g + i] * sc);
      *(bf16x4*)((uint16_t*)a.dQ + base + (size_t)q * DH + 32 * (2 * dh + j) + 8 * g + 4 * h) = v;
    }
}

// ============================================================== dispatch
static bool mfma_ok(int Dh, int dt, const void* O, int ld_o) {
  return Dh == DH && dt == BF16 && ((uintptr_t)O % 16 == 0) && (ld_o % 8 == 0);
}

int attention_fwd_mfma(const AttnFwd& a, hipStream_t s) {
  if (!mfma_ok(a.Dh, a.dt, a.O, a.ld_o)) return -1;
  dim3 grid((a.N + F_QB - 1) / F_QB, a.B * a.H);
  const double nn = (double)a.B * a.H * a.N * (double)a.N * DH;
  const int pi = prof_begin(PROF_ATTN_FWD);
  // the direct-load kernel addresses K and V with 32-bit byte offsets
  if ((double)a.N * DH * 2.0 * 3 < 2147483000.0)
    launch(attn_fwd2_k, dim3((a.N + F2_QB - 1) / F2_QB, a.B * a.H), dim3(256), 0u, s, a);
  else
    launch(attn_fwd_mfma_k, grid, dim3(256), 0u, s, a);
  prof_end(pi, 4.0 * nn);
  JG_CHECK_LAUNCH("attention_fwd_mfma");
  return 0;
}

int attention_bwd_mfma(const AttnBwd& a, hipStream_t s) {
  if (!mfma_ok(a.Dh, a.dt, a.dO, a.ld_do) || a.dt_d != BF16 || (uintptr_t)a.O % 16 || a.ld_o % 8) return -1;
  hipLaunchKernelGGL(attn_delta_mfma_k, dim3((a.rm.rows() + 3) / 4), dim3(256), 0, s, a);
  JG_CHECK_LAUNCH("attention_delta_mfma");
  const double nn = (double)a.B * a.H * a.N * (double)a.N * DH;
  // the direct-load kernels address dO with 32-bit byte offsets
  const bool v2 = (double)a.rm.rows() * a.ld_do * 2.0 < 2147483000.0 && (double)a.N * DH * 2.0 * 3 < 2147483000.0;
  // stored dS^T: the geometry the kernels assume, and 32-bit offsets per head
  // (the dQ pass fetches up to four key tiles past the padded count)
  const bool ds = a.dS && a.nk_pad == attn_ds_rows(a.N) && a.ld_ds == attn_ds_ld(a.N) &&
                  (double)(a.nk_pad + 512) * a.ld_ds * 2.0 < 2147483000.0 && (uintptr_t)a.dS % 16 == 0;
  AttnBwd ak = a;
  if (!ds) ak.dS = nullptr;
  int pi = prof_begin(PROF_ATTN_BWD_KV);
  if (v2 && ds) launch(attn_bwd_kv5_k<true>, dim3((a.N + KV5_KB - 1) / KV5_KB, a.B * a.H), dim3(512), 0u, s, ak);
  else if (v2) launch(attn_bwd_kv5_k<false>, dim3((a.N + KV5_KB - 1) / KV5_KB, a.B * a.H), dim3(512), 0u, s, ak);
  else launch(attn_bwd_kv_mfma_k, dim3((a.N + KV_KB - 1) / KV_KB, a.B * a.H), dim3(256), 0u, s, a);
  prof_end(pi, 6.0 * nn);
  JG_CHECK_LAUNCH("attention_bwd_kv_mfma");
  pi = prof_begin(PROF_ATTN_BWD_Q);
  if (v2 && ds) launch(attn_bwd_q4_k, dim3((a.N + Q4_QB - 1) / Q4_QB, a.B * a.H), dim3(512), 0u, s, a);
  else if (v2) launch(attn_bwd_q2_k, dim3((a.N + Q2_QB - 1) / Q2_QB, a.B * a.H), dim3(256), 0u, s, a);
  else launch(attn_bwd_q_mfma_k, dim3((a.N + Q_QB - 1) / Q_QB, a.B * a.H), dim3(256), 0u, s, a);
  prof_end(pi, 2.0 * nn);
  JG_CHECK_LAUNCH("attention_bwd_q_mfma");
  return 0;
}

}  // namespace jg
