// GEMMs of the DiT forward and backward on gfx950.
//
// bf16 operands go through an LDS-tiled MFMA kernel (v_mfma_f32_32x32x16_bf16,
// fp32 accumulation).  Both operands are staged in LDS in one canonical layout,
// "row x k, k contiguous", so that every MFMA fragment is one 16-byte LDS read.
// An operand whose contraction index is the strided one (the token-row
// contraction of the weight gradients, the weight operand of the input
// gradients) is fetched as 8x8 element blocks with 16-byte global loads and
// transposed in registers before the LDS write, instead of being re-laid out in
// HBM by a separate pass.
//
// Workgroup -> tile mapping is XCD-aware: the hardware deals workgroups to the
// 8 XCDs round-robin, so consecutive tile ids are first regrouped per XCD and
// then walked in GROUP_M-row bands, keeping the A rows and B columns a band
// shares in one XCD's L2.
//
// Anything else (fp32 operands, contiguous dims not multiple of 8) takes a
// plain LDS-tiled VALU kernel with fp32 accumulation.
#include "gemm.h"
#include "prof.h"

namespace jg {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ inline void epi_apply(const Epi& e, int r, int c, float v) {
  if (e.bias) v += ld_any(e.bias, e.bias_dt, c);
  if (e.mode == EPI_GELU_FWD) {
    st_any(e.aux, e.aux_dt, (size_t)r * e.ldaux + c, v);
    v = gelu_tanh(v);
  } else if (e.mode == EPI_GELU_BWD) {
    v *= gelu_tanh_grad(ld_any(e.aux, e.aux_dt, (size_t)r * e.ldaux + c));
  }
  const size_t idx = (size_t)r * e.ldc + c;
  if (e.beta != 0.f) v += e.beta * ld_any(e.C, e.c_dt, idx);
  st_any(e.C, e.c_dt, idx, v);
}

__device__ inline int xcd_remap(int b, int total) {
  const int per = total / 8, rem = total % 8;
  const int xcd = b % 8, local = b / 8;
  return xcd < rem ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
}

__device__ inline void tile_coords(int id, int tiles_m, int tiles_n, int& tm, int& tn) {
  constexpr int GROUP_M = 8;
  const int in_group = GROUP_M * tiles_n;
  const int gid = id / in_group;
  const int first = gid * GROUP_M;
  const int gsz = min(tiles_m - first, GROUP_M);
  const int r = id % in_group;
  tm = first + r % gsz;
  tn = r / gsz;
}

// ------------------------------------------------------------ tile loaders
// Loads a ROWS x BK tile of an operand into registers and stores it into LDS
// as S[row * LDSK + k].
template <int ROWS, int BK, int NT, bool T>
struct Loader;

template <int ROWS, int BK, int NT>
struct Loader<ROWS, BK, NT, false> {  // P[row * ld + k], vectors along k
  static constexpr int NVEC = ROWS * BK / 8;
  static constexpr int NV = (NVEC + NT - 1) / NT;
  u32x4 r[NV];
  __device__ inline void load(const uint16_t* P, int ld, int row0, int nrows, int k0, int K) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int v = threadIdx.x + i * NT;
      const int row = v / (BK / 8), kv = v % (BK / 8);
      const int gr = row0 + row, gk = k0 + kv * 8;
      if (v < NVEC && gr < nrows && gk < K)
        r[i] = *(const u32x4*)(P + (size_t)gr * ld + gk);
      else
        r[i] = u32x4{0u, 0u, 0u, 0u};
    }
  }
  template <int LDSK>
  __device__ inline void store(uint16_t* S) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int v = threadIdx.x + i * NT;
      if (v < NVEC) {
        const int row = v / (BK / 8), kv = v % (BK / 8);
        *(u32x4*)(S + row * LDSK + kv * 8) = r[i];
      }
    }
  }
};

template <int ROWS, int BK, int NT>
struct Loader<ROWS, BK, NT, true> {  // P[k * ld + row], 8x8 blocks transposed in registers
  static constexpr int NBLK = (ROWS / 8) * (BK / 8);
  static constexpr int NB = (NBLK + NT - 1) / NT;
  u32x4 r[NB * 8];
  __device__ inline void load(const uint16_t* P, int ld, int row0, int nrows, int k0, int K) {
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int b = threadIdx.x + i * NT;
      const int kb = b / (ROWS / 8), rb = b % (ROWS / 8);
      const int gr = row0 + rb * 8;
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) {
        const int gk = k0 + kb * 8 + kk;
        if (b < NBLK && gr < nrows && gk < K)
          r[i * 8 + kk] = *(const u32x4*)(P + (size_t)gk * ld + gr);
        else
          r[i * 8 + kk] = u32x4{0u, 0u, 0u, 0u};
      }
    }
  }
  template <int LDSK>
  __device__ inline void store(uint16_t* S) {
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int b = threadIdx.x + i * NT;
      if (b >= NBLK) continue;
      const int kb = b / (ROWS / 8), rb = b % (ROWS / 8);
      const u32x4* in = r + i * 8;
      // out[m] word w = element (k=2w, m) | element (k=2w+1, m) << 16
#pragma unroll
      for (int mw = 0; mw < 4; ++mw) {  // rows m = 2mw (low halves) and 2mw+1 (high halves)
        u32x4 lo, hi;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const unsigned a = in[2 * w][mw], c = in[2 * w + 1][mw];
          lo[w] = (a & 0xffffu) | (c << 16);
          hi[w] = (a >> 16) | (c & 0xffff0000u);
        }
        *(u32x4*)(S + (rb * 8 + 2 * mw) * LDSK + kb * 8) = lo;
        *(u32x4*)(S + (rb * 8 + 2 * mw + 1) * LDSK + kb * 8) = hi;
      }
    }
  }
};

// --------------------------------------------------------------- MFMA GEMM
template <int BM, int BN, int BK, int WM, int WN, bool TA, bool TB>
__global__ __launch_bounds__(WM * WN * 64) void gemm_mfma_kernel(GemmArgs g) {
  constexpr int NT = WM * WN * 64;
  constexpr int LDSK = BK + 8;
  constexpr int TMW = BM / WM, TNW = BN / WN;
  constexpr int FM = TMW / 32, FN = TNW / 32;
  __shared__ __attribute__((aligned(16))) uint16_t As[BM * LDSK];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[BN * LDSK];

  const int tiles_m = (g.M + BM - 1) / BM, tiles_n = (g.N + BN - 1) / BN;
  int tm, tn;
  tile_coords(xcd_remap(blockIdx.x, tiles_m * tiles_n), tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;

  Loader<BM, BK, NT, TA> la;
  Loader<BN, BK, NT, TB> lb;
  const uint16_t* A = (const uint16_t*)g.A;
  const uint16_t* B = (const uint16_t*)g.B;

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  const int nk = (g.K + BK - 1) / BK;
  la.load(A, g.lda, m0, g.M, 0, g.K);
  lb.load(B, g.ldb, n0, g.N, 0, g.K);
  for (int kt = 0; kt < nk; ++kt) {
    __syncthreads();
    la.template store<LDSK>(As);
    lb.template store<LDSK>(Bs);
    __syncthreads();
    if (kt + 1 < nk) {
      la.load(A, g.lda, m0, g.M, (kt + 1) * BK, g.K);
      lb.load(B, g.ldb, n0, g.N, (kt + 1) * BK, g.K);
    }
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      bf16x8 a[FM], b[FN];
      const int ko = kk * 16 + (lane >> 5) * 8;
#pragma unroll
      for (int i = 0; i < FM; ++i)
        a[i] = __builtin_bit_cast(bf16x8, *(const u32x4*)(As + (wm * TMW + i * 32 + (lane & 31)) * LDSK + ko));
#pragma unroll
      for (int j = 0; j < FN; ++j)
        b[j] = __builtin_bit_cast(bf16x8, *(const u32x4*)(Bs + (wn * TNW + j * 32 + (lane & 31)) * LDSK + ko));
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  }

  // 32x32 accumulator layout: lane holds column (lane % 32); register e holds
  // row 8*(e/4) + 4*(lane/32) + e%4.
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int col = n0 + wn * TNW + j * 32 + (lane & 31);
      if (col >= g.N) continue;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = m0 + wm * TMW + i * 32 + (e >> 2) * 8 + (lane >> 5) * 4 + (e & 3);
        if (row < g.M) epi_apply(g.epi, row, col, acc[i][j][e]);
      }
    }
}

// ---------------------------------------------------------------- VALU GEMM
// 64x64 tile, 256 threads, 4x4 outputs per thread, fp32 accumulation, any
// layout and operand dtype.
__global__ __launch_bounds__(256) void gemm_valu_kernel(GemmArgs g) {
  constexpr int T = 64, KT = 16;
  __shared__ float As[KT][T + 1];
  __shared__ float Bs[KT][T + 1];
  const int m0 = blockIdx.y * T, n0 = blockIdx.x * T;
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < g.K; k0 += KT) {
    for (int i = threadIdx.x; i < KT * T; i += 256) {
      const int kk = i / T, mm = i % T;
      const int k = k0 + kk;
      const int m = m0 + mm, n = n0 + mm;
      float a = 0.f, b = 0.f;
      if (k < g.K && m < g.M)
        a = ld_any(g.A, g.a_dt, g.ta ? (size_t)k * g.lda + m : (size_t)m * g.lda + k);
      if (k < g.K && n < g.N)
        b = ld_any(g.B, g.b_dt, g.tb ? (size_t)k * g.ldb + n : (size_t)n * g.ldb + k);
      As[kk][mm] = a;
      Bs[kk][mm] = b;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < KT; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = As[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = Bs[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + ty + 16 * i, n = n0 + tx + 16 * j;
      if (m < g.M && n < g.N) epi_apply(g.epi, m, n, acc[i][j]);
    }
}

// ------------------------------------------------------------------ launch
template <int BM, int BN, int BK, int WM, int WN, bool TA, bool TB>
static int launch_mfma(const GemmArgs& g, hipStream_t s) {
  const int tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  hipLaunchKernelGGL((gemm_mfma_kernel<BM, BN, BK, WM, WN, TA, TB>), dim3(tiles), dim3(WM * WN * 64), 0, s, g);
  JG_CHECK_LAUNCH("gemm_mfma");
  return 0;
}

static int prof_class(const GemmArgs& g) {
  if (!g.ta && !g.tb) return PROF_GEMM_FWD;
  if (!g.ta && g.tb) return PROF_GEMM_DGRAD;
  if (g.ta && g.tb) return PROF_GEMM_WGRAD;
  return PROF_NONE;
}

static int gemm_launch(const GemmArgs& g, hipStream_t s);

int gemm(const GemmArgs& g, hipStream_t s) {
  const int pi = prof_begin(prof_class(g), s);
  const int rc = gemm_launch(g, s);
  prof_end(pi, s, 2.0 * g.M * g.N * (double)g.K);
  return rc;
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

static int gemm_launch(const GemmArgs& g, hipStream_t s) {
  if (g.M < 0 || g.N < 0 || g.K < 0 || !g.A || !g.B || !g.epi.C) {
    set_error("gemm: invalid arguments");
    return 1;
  }
  if (g.M == 0 || g.N == 0) return 0;
  bool mfma = g.a_dt == BF16 && g.b_dt == BF16 && g.K > 0 && aligned16(g.A) && aligned16(g.B) &&
              g.lda % 8 == 0 && g.ldb % 8 == 0;
  if (mfma) mfma = (g.ta ? g.M % 8 == 0 : g.K % 8 == 0) && (g.tb ? g.N % 8 == 0 : g.K % 8 == 0);
  if (mfma) {
    if (!g.ta && !g.tb) return launch_mfma<128, 128, 64, 2, 2, false, false>(g, s);
    if (!g.ta && g.tb) return launch_mfma<128, 128, 64, 2, 2, false, true>(g, s);
    if (g.ta && g.tb) return launch_mfma<128, 128, 64, 2, 2, true, true>(g, s);
    return launch_mfma<128, 128, 64, 2, 2, true, false>(g, s);
  }
  dim3 grid((g.N + 63) / 64, (g.M + 63) / 64);
  if (g.K == 0) {
    // an empty contraction still applies the epilogue (bias, beta)
  }
  hipLaunchKernelGGL(gemm_valu_kernel, grid, dim3(256), 0, s, g);
  JG_CHECK_LAUNCH("gemm_valu");
  return 0;
}

}  // namespace jg
