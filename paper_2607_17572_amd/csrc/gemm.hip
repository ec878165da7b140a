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
#include <atomic>
#include "gemm.h"
#include <type_traits>
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
// Operands are read through buffer resources: an out-of-range offset returns
// zero, so ragged edges cost a select per load instead of a branch.
constexpr int OOB = 0x7ffffff0;

__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* p, long bytes) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)p, (short)0, (int)bytes, 0x00020000);
}
__device__ inline u32x4 bload(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

// Loads a ROWS x BK tile of an operand into registers and stores it into LDS
// as S[row * LDSK + k].
template <int ROWS, int BK, int NT, bool T>
struct Loader;

template <int ROWS, int BK, int NT>
struct Loader<ROWS, BK, NT, false> {  // P[row * ld + k], vectors along k
  static constexpr int NVEC = ROWS * BK / 8;
  static constexpr int NV = (NVEC + NT - 1) / NT;
  u32x4 r[NV];
  __device__ inline void load(__amdgpu_buffer_rsrc_t P, int ld, int row0, int nrows, int k0, int K) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int v = threadIdx.x + i * NT;
      const int row = v / (BK / 8), kv = v % (BK / 8);
      const int gr = row0 + row, gk = k0 + kv * 8;
      const bool ok = (NVEC % NT == 0 || v < NVEC) && gr < nrows && gk < K;
      r[i] = bload(P, ok ? (gr * ld + gk) * 2 : OOB);
    }
  }
  template <int LDSK>
  __device__ inline void store(uint16_t* S) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int v = threadIdx.x + i * NT;
      if (NVEC % NT == 0 || v < NVEC) {
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
  __device__ inline void load(__amdgpu_buffer_rsrc_t P, int ld, int row0, int nrows, int k0, int K) {
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int b = threadIdx.x + i * NT;
      // lanes vary the k block fastest: the 16 lanes of a 16-byte LDS store
      // group then cover 8 k blocks x 2 row parities = 16 distinct bank groups
      const int kb = b % (BK / 8), rb = b / (BK / 8);
      const int gr = row0 + rb * 8;
      const bool okb = (NBLK % NT == 0 || b < NBLK) && gr < nrows;
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) {
        const int gk = k0 + kb * 8 + kk;
        r[i * 8 + kk] = bload(P, (okb && gk < K) ? (gk * ld + gr) * 2 : OOB);
      }
    }
  }
  template <int LDSK>
  __device__ inline void store(uint16_t* S) {
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int b = threadIdx.x + i * NT;
      if (NBLK % NT != 0 && b >= NBLK) continue;
      const int kb = b % (BK / 8), rb = b / (BK / 8);
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

// ------------------------------------------------------------ epilogues
// Output kinds (the host picks one per launch):
enum EpiKind {
  EK_F32 = 0,       // C fp32 = acc
  EK_F32_ACC = 1,   // C fp32 += acc
  EK_BF16 = 2,      // C bf16 = acc
  EK_BF16_ACC = 3,  // C bf16 += acc
  EK_BIAS = 4,      // C bf16 = acc + bias
  EK_GELU = 5,      // aux bf16 = acc + bias, C bf16 = gelu(aux)
  EK_DGELU = 6,     // C bf16 = acc * gelu'(aux)
};

__device__ __forceinline__ void unpack8(const u32x4& u, float* f) {
#pragma unroll
  for (int w = 0; w < 4; ++w) { f[2 * w] = bf2f(u[w] & 0xffffu); f[2 * w + 1] = bf2f(u[w] >> 16); }
}
__device__ __forceinline__ u32x4 pack8(const float* f) {
  u32x4 u;
#pragma unroll
  for (int w = 0; w < 4; ++w) u[w] = (uint32_t)f2bf(f[2 * w]) | ((uint32_t)f2bf(f[2 * w + 1]) << 16);
  return u;
}

// 8 consecutive outputs of one row, all inside C (vector path)
template <int EK>
__device__ __forceinline__ void epi8(const Epi& e, int row, int col, float* v) {
  if (EK == EK_BIAS || EK == EK_GELU) {
    float bb[8];
    unpack8(*(const u32x4*)((const uint16_t*)e.bias + col), bb);
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] += bb[q];
  }
  if (EK == EK_GELU) {
    *(u32x4*)((uint16_t*)e.aux + (size_t)row * e.ldaux + col) = pack8(v);
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = gelu_tanh(v[q]);
  }
  if (EK == EK_DGELU) {
    float pa[8];
    unpack8(*(const u32x4*)((const uint16_t*)e.aux + (size_t)row * e.ldaux + col), pa);
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] *= gelu_tanh_grad(pa[q]);
  }
  if (EK == EK_F32 || EK == EK_F32_ACC) {
    float4* cp = (float4*)((float*)e.C + (size_t)row * e.ldc + col);
#pragma unroll
    for (int w = 0; w < 2; ++w) {
      float4 x = make_float4(v[4 * w], v[4 * w + 1], v[4 * w + 2], v[4 * w + 3]);
      if (EK == EK_F32_ACC) {
        const float4 o = cp[w];
        x.x += o.x; x.y += o.y; x.z += o.z; x.w += o.w;
      }
      cp[w] = x;
    }
  } else {
    uint16_t* cp = (uint16_t*)e.C + (size_t)row * e.ldc + col;
    if (EK == EK_BF16_ACC) {
      float o[8];
      unpack8(*(const u32x4*)cp, o);
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] += o[q];
    }
    *(u32x4*)cp = pack8(v);
  }
}

// one output element (edge path)
template <int EK>
__device__ __forceinline__ void epi1(const Epi& e, int row, int col, float v) {
  if (EK == EK_BIAS || EK == EK_GELU) v += bf2f(((const uint16_t*)e.bias)[col]);
  if (EK == EK_GELU) {
    ((uint16_t*)e.aux)[(size_t)row * e.ldaux + col] = f2bf(v);
    v = gelu_tanh(v);
  }
  if (EK == EK_DGELU) v *= gelu_tanh_grad(bf2f(((const uint16_t*)e.aux)[(size_t)row * e.ldaux + col]));
  const size_t idx = (size_t)row * e.ldc + col;
  if (EK == EK_F32 || EK == EK_F32_ACC) {
    float* cp = (float*)e.C;
    cp[idx] = (EK == EK_F32_ACC ? cp[idx] : 0.f) + v;
  } else {
    uint16_t* cp = (uint16_t*)e.C;
    cp[idx] = f2bf((EK == EK_BF16_ACC ? bf2f(cp[idx]) : 0.f) + v);
  }
}

// Epilogue of the MFMA kernels.  Accumulator layout: lane holds column
// (lane % 32), register e holds row 8*(e/4) + 4*(lane/32) + e%4.  Each 32x32
// tile is staged transposed through LDS (T[col][row], stride 36 floats) so that
// every lane then owns 16 consecutive outputs of one row.
template <int BM, int BN, int WM, int WN, int EK>
__device__ __forceinline__ void mfma_epilogue(const GemmArgs& g, f32x16 (&acc)[BM / WM / 32][BN / WN / 32], int m0, int n0,
                                     uint16_t* lds) {
  constexpr int TMW = BM / WM, TNW = BN / WN;
  constexpr int FM = TMW / 32, FN = TNW / 32;
  constexpr int ES = 36;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
  float* T = (float*)lds + wave * 32 * ES;
  const int h = lane >> 5, c32 = lane & 31;
  const int rr = lane >> 1, cc = (lane & 1) * 16;
  const bool vec_ok = (g.N % 8 == 0) && (g.epi.ldc % 8 == 0);
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        float4 x = make_float4(acc[i][j][4 * gq], acc[i][j][4 * gq + 1], acc[i][j][4 * gq + 2], acc[i][j][4 * gq + 3]);
        *(float4*)(T + c32 * ES + 8 * gq + 4 * h) = x;
      }
      __syncthreads();
      const int row = m0 + wm * TMW + i * 32 + rr;
      // kept rolled: the accumulator tiles above must stay fully unrolled
      // (static register indices), and the whole epilogue has to fit the
      // unroller's budget for that
#pragma unroll 1
      for (int half = 0; half < 2; ++half) {
        float v[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] = T[(cc + 8 * half + q) * ES + rr];
        const int col = n0 + wn * TNW + j * 32 + cc + 8 * half;
        if (row < g.M) {
          if (vec_ok && col + 8 <= g.N) {
            epi8<EK>(g.epi, row, col, v);
          } else {
#pragma unroll 1
            for (int q = 0; q < 8; ++q)
              if (col + q < g.N) epi1<EK>(g.epi, row, col + q, T[(cc + 8 * half + q) * ES + rr]);
          }
        }
      }
      __syncthreads();
    }
}

// --------------------------------------------------------------- MFMA GEMM
// BM x BN workgroup tile, WM x WN waves (each (BM/WM) x (BN/WN), made of 32x32
// MFMA tiles), BK-deep k steps through two LDS stages: the global loads of
// step k+1 are in flight while step k's MFMAs run, and one barrier per step
// separates the LDS write of the next stage from the reads of the current one.
// The epilogue stages each 32x32 accumulator tile through LDS (transposed) so
// that every lane then owns 16 consecutive outputs of one row: 16-byte
// global stores and vector reads of bias / GELU input / the accumulated C.
template <int BM, int BN, int BK, int WM, int WN, bool TA, bool TB, int EK>
__global__ __launch_bounds__(WM * WN * 64) void gemm_mfma_kernel(GemmArgs g) {
  constexpr int NT = WM * WN * 64;
  constexpr int LDSK = BK + 8;
  constexpr int TMW = BM / WM, TNW = BN / WN;
  constexpr int FM = TMW / 32, FN = TNW / 32;
  constexpr int STAGE = (BM + BN) * LDSK;
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];

  const int tiles_m = (g.M + BM - 1) / BM, tiles_n = (g.N + BN - 1) / BN;
  int tm, tn;
  tile_coords(xcd_remap(blockIdx.x, tiles_m * tiles_n), tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;

  Loader<BM, BK, NT, TA> la;
  Loader<BN, BK, NT, TB> lb;
  const long ext_a = TA ? ((long)(g.K - 1) * g.lda + g.M) * 2 : ((long)(g.M - 1) * g.lda + g.K) * 2;
  const long ext_b = TB ? ((long)(g.K - 1) * g.ldb + g.N) * 2 : ((long)(g.N - 1) * g.ldb + g.K) * 2;
  const __amdgpu_buffer_rsrc_t RA = make_rsrc(g.A, ext_a), RB = make_rsrc(g.B, ext_b);

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  // Pipeline: LDS holds tiles kt (being read) and kt+1 (written at the top of
  // iteration kt from registers); the registers receive tile kt+2, so every
  // global load has a full iteration of MFMA work to land.
  const int nk = (g.K + BK - 1) / BK;
  la.load(RA, g.lda, m0, g.M, 0, g.K);
  lb.load(RB, g.ldb, n0, g.N, 0, g.K);
  la.template store<LDSK>(lds);
  lb.template store<LDSK>(lds + BM * LDSK);
  if (nk > 1) {
    la.load(RA, g.lda, m0, g.M, BK, g.K);
    lb.load(RB, g.ldb, n0, g.N, BK, g.K);
  }
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const uint16_t* As = lds + (kt & 1) * STAGE;
    const uint16_t* Bs = As + BM * LDSK;
    if (kt + 1 < nk) {
      uint16_t* An = lds + ((kt + 1) & 1) * STAGE;
      la.template store<LDSK>(An);
      lb.template store<LDSK>(An + BM * LDSK);
    }
    if (kt + 2 < nk) {
      la.load(RA, g.lda, m0, g.M, (kt + 2) * BK, g.K);
      lb.load(RB, g.ldb, n0, g.N, (kt + 2) * BK, g.K);
    }
    // fragments of step kk+1 are read from LDS while the MFMAs of step kk run
    constexpr int KS = BK / 16;
    bf16x8 fa[2][FM], fb[2][FN];
    auto ldfrag = [&](int kk, int buf) {
      const int ko = kk * 16 + (lane >> 5) * 8;
#pragma unroll
      for (int i = 0; i < FM; ++i)
        fa[buf][i] = __builtin_bit_cast(bf16x8, *(const u32x4*)(As + (wm * TMW + i * 32 + (lane & 31)) * LDSK + ko));
#pragma unroll
      for (int j = 0; j < FN; ++j)
        fb[buf][j] = __builtin_bit_cast(bf16x8, *(const u32x4*)(Bs + (wn * TNW + j * 32 + (lane & 31)) * LDSK + ko));
    };
    ldfrag(0, 0);
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const int cb = kk & 1;
      if (kk + 1 < KS) ldfrag(kk + 1, cb ^ 1);
      // keep the reads of step kk+1 ahead of the MFMAs of step kk
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[cb][i], fb[cb][j], acc[i][j], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
  }

  __syncthreads();
  mfma_epilogue<BM, BN, WM, WN, EK>(g, acc, m0, n0, lds);
}

// ------------------------------------------------- pipelined MFMA GEMM
// For K a multiple of 64.  Same tiles, LDS layout and epilogue as above, but
// the k loop is software-pipelined at the instruction level: every 16-deep
// MFMA step issues, between its MFMAs, the LDS fragment reads of the next step,
// a share of the LDS writes of the next k tile and the global loads of the one
// after (sched_group_barrier fixes that interleave), and the workgroup barrier
// sits before the last MFMA step of a tile so that step hides the first
// fragment reads of the next tile.
//
// All global offsets go through the per-lane voffset of a buffer resource, so
// the hardware range check covers them: loads past the end of an operand (the
// two tiles fetched beyond K at the end of the loop, rows past M or N in the
// last row of an operand) return zero or in-buffer data that only reaches
// outputs that are never stored.
__device__ inline u32x4 bload_v(__amdgpu_buffer_rsrc_t r, int voff) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, 0, 0));
}

// k-contiguous operand, P[row * ld + k]: NV 16-byte vectors per thread, RSTEP
// rows apart, in NSET register sets (a set is refilled right after its
// contents went to LDS, so NSET sets give the loads NSET k tiles to land);
// load / store a part [LO, HI) of the vectors per call.
template <int ROWS, int BK, int NT, int LDSK, int NSET>
struct PipeN {
  static constexpr int VPR = BK / 8;
  static constexpr int NV = ROWS * VPR / NT;
  static constexpr int RSTEP = NT / VPR;
  static_assert(ROWS * VPR % NT == 0 && NV >= 1, "tile rows x k must split evenly over the threads");
  static constexpr int NS = NV;  // store units (one 16-byte LDS write each)
  u32x4 r[NSET][NV];
  int voff, sidx, step;
  __device__ inline void init(int ld, int row0) {
    const int row = threadIdx.x / VPR, kv = threadIdx.x % VPR;
    voff = ((row0 + row) * ld + kv * 8) * 2;
    sidx = row * LDSK + kv * 8;
    step = RSTEP * ld * 2;
  }
  template <int SET, int LO, int HI>
  __device__ inline void load(__amdgpu_buffer_rsrc_t R, int k0) {
#pragma unroll
    for (int i = LO; i < HI; ++i) r[SET][i] = bload_v(R, voff + (k0 * 2 + i * step));
  }
  template <int SET, int LO, int HI>
  __device__ inline void store(uint16_t* S) const {
#pragma unroll
    for (int i = LO; i < HI; ++i) *(u32x4*)(S + sidx + i * RSTEP * LDSK) = r[SET][i];
  }
};

// k-strided operand, P[k * ld + row]: one 8x8 block per thread (threads past
// the block count repeat a block: same data to the same place), transposed in
// registers with byte permutes.
template <int ROWS, int BK, int NT, int LDSK, int NSET>
struct PipeT {
  static constexpr int KB = BK / 8, NBLK = (ROWS / 8) * KB;
  static constexpr int NB = NBLK > NT ? NBLK / NT : 1;
  static_assert(NBLK % NT == 0 || NT % NBLK == 0, "8x8 blocks must split evenly over the threads");
  static constexpr int NV = NB * 8;  // loads
  static constexpr int NS = NB * 4;  // store units (two 16-byte LDS writes each)
  u32x4 r[NSET][NB * 8];
  int voff[NB], sidx[NB];
  int ld2;
  __device__ inline void init(int ld, int row0) {
    ld2 = ld * 2;
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int b = (threadIdx.x + i * NT) % NBLK;
      const int kb = b % KB, rb = b / KB;  // k block fastest: conflict-free 16-byte LDS writes
      voff[i] = (kb * 8 * ld + row0 + rb * 8) * 2;
      sidx[i] = rb * 8 * LDSK + kb * 8;
    }
  }
  template <int SET, int LO, int HI>
  __device__ inline void load(__amdgpu_buffer_rsrc_t R, int k0) {
#pragma unroll
    for (int v = LO; v < HI; ++v) r[SET][v] = bload_v(R, voff[v / 8] + (k0 + v % 8) * ld2);
  }
  // unit u = (block u / 4, row pair u % 4): rows m = 2mw, 2mw+1 of the block,
  // word w = element (k = 2w, m) | element (k = 2w + 1, m) << 16
  template <int SET, int LO, int HI>
  __device__ inline void store(uint16_t* S) const {
#pragma unroll
    for (int u = LO; u < HI; ++u) {
      const int i = u / 4, mw = u % 4;
      const u32x4* in = r[SET] + i * 8;
      u32x4 lo, hi;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        lo[w] = __builtin_amdgcn_perm(in[2 * w + 1][mw], in[2 * w][mw], 0x05040100u);
        hi[w] = __builtin_amdgcn_perm(in[2 * w + 1][mw], in[2 * w][mw], 0x07060302u);
      }
      *(u32x4*)(S + sidx[i] + (2 * mw) * LDSK) = lo;
      *(u32x4*)(S + sidx[i] + (2 * mw + 1) * LDSK) = hi;
    }
  }
};

template <bool T, int ROWS, int BK, int NT, int LDSK, int NSET>
struct PipeSel { typedef PipeN<ROWS, BK, NT, LDSK, NSET> type; };
template <int ROWS, int BK, int NT, int LDSK, int NSET>
struct PipeSel<true, ROWS, BK, NT, LDSK, NSET> { typedef PipeT<ROWS, BK, NT, LDSK, NSET> type; };

// Instruction interleave of one MFMA step: MF MFMAs, with R LDS reads, W LDS
// writes and L global loads dealt out between them (reads and writes
// alternating, then loads), in that order.
template <int O, int HI, int R, int W>
__device__ __forceinline__ void sched_ops() {
  if constexpr (O < HI) {
    constexpr int RW = 2 * (R < W ? R : W);
    constexpr int kind = O < RW ? O % 2 : (O < R + W ? (R > W ? 0 : 1) : 2);
    __builtin_amdgcn_sched_group_barrier(kind == 0 ? 0x100 : (kind == 1 ? 0x200 : 0x020), 1, 0);
    sched_ops<O + 1, HI, R, W>();
  }
}
template <int MF, int R, int W, int L, int I = 0>
__device__ __forceinline__ void pipe_sched() {
  if constexpr (I < MF) {
    constexpr int T = R + W + L;
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    sched_ops<I * T / MF, (I + 1) * T / MF, R, W>();
    pipe_sched<MF, R, W, L, I + 1>();
  }
}

template <int BM, int BN, int BK, int WM, int WN, bool TA, bool TB, int EK>
__global__ __launch_bounds__(WM * WN * 64) void gemm_pipe_kernel(GemmGroup gg) {
  static_assert(BK == 64, "the schedule is written for four 16-deep MFMA steps per k tile");
  constexpr int NT = WM * WN * 64;
  constexpr int LDSK = BK + 8;
  constexpr int TMW = BM / WM, TNW = BN / WN;
  constexpr int FM = TMW / 32, FN = TNW / 32;
  constexpr int STAGE = (BM + BN) * LDSK;
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];

  // the first tiles0 workgroups compute problem 0, the rest problem 1
  const int sel = (int)blockIdx.x >= gg.tiles0 ? 1 : 0;
  const GemmArgs& g = gg.p[sel];
  const int local = (int)blockIdx.x - sel * gg.tiles0;
  const int tiles_m = (g.M + BM - 1) / BM, tiles_n = (g.N + BN - 1) / BN;
  int tm, tn;
  tile_coords(xcd_remap(local, tiles_m * tiles_n), tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;

  // 4-wave tiles keep two register sets (loads two k tiles ahead); 8-wave
  // tiles have half the registers per wave and keep one
  constexpr int NSET = NT == 256 ? 2 : 1;
  typedef typename PipeSel<TA, BM, BK, NT, LDSK, NSET>::type LA;
  typedef typename PipeSel<TB, BN, BK, NT, LDSK, NSET>::type LB;
  LA la;
  LB lb;
  la.init(g.lda, m0);
  lb.init(g.ldb, n0);
  const long ext_a = TA ? ((long)(g.K - 1) * g.lda + g.M) * 2 : ((long)(g.M - 1) * g.lda + g.K) * 2;
  const long ext_b = TB ? ((long)(g.K - 1) * g.ldb + g.N) * 2 : ((long)(g.N - 1) * g.ldb + g.K) * 2;
  const __amdgpu_buffer_rsrc_t RA = make_rsrc(g.A, ext_a), RB = make_rsrc(g.B, ext_b);

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  const int fro = (lane & 31) * LDSK + (lane >> 5) * 8;  // this lane's fragment offset
  bf16x8 fa[2][FM], fb[2][FN];
  auto ldfrag = [&](const uint16_t* S, int kk, int buf) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
      fa[buf][i] = __builtin_bit_cast(bf16x8, *(const u32x4*)(S + (wm * TMW + i * 32) * LDSK + fro + kk * 16));
#pragma unroll
    for (int j = 0; j < FN; ++j)
      fb[buf][j] = __builtin_bit_cast(bf16x8, *(const u32x4*)(S + (BM + wn * TNW + j * 32) * LDSK + fro + kk * 16));
  };
  auto mfma_step = [&](int buf) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[buf][i], fb[buf][j], acc[i][j], 0, 0, 0);
  };

  // prologue: tile 0 into LDS stage 0; tiles 1 .. NSET into the register sets
  // (tile t lives in set t % NSET)
  la.template load<0, 0, LA::NV>(RA, 0);
  lb.template load<0, 0, LB::NV>(RB, 0);
  if constexpr (NSET == 2) {
    la.template load<1, 0, LA::NV>(RA, BK);
    lb.template load<1, 0, LB::NV>(RB, BK);
  }
  la.template store<0, 0, LA::NS>(lds);
  lb.template store<0, 0, LB::NS>(lds + BM * LDSK);
  la.template load<0, 0, LA::NV>(RA, NSET * BK);
  lb.template load<0, 0, LB::NV>(RB, NSET * BK);
  __syncthreads();
  ldfrag(lds, 0, 0);

  // Per k tile kt: stage kt&1 is read, stage (kt+1)&1 is written from register
  // set (kt+1) % NSET, which is then refilled with tile kt+1+NSET:
  //   k-contiguous operand: its vectors stored and reloaded in thirds over
  //     MFMA steps 0, 1, 2;
  //   k-strided operand: A's block stored and reloaded in step 0, B's in step 1.
  constexpr int MF = FM * FN, RD = FM + FN;
  constexpr int A1 = LA::NV / 3, A2 = 2 * LA::NV / 3, B1 = LB::NV / 3, B2 = 2 * LB::NV / 3;
  constexpr int WA0 = TA ? 2 * LA::NS : A1, WA1 = TA ? 0 : A2 - A1, WA2 = TA ? 0 : LA::NV - A2;
  constexpr int LA0 = TA ? LA::NV : A1, LA1 = TA ? 0 : A2 - A1, LA2 = TA ? 0 : LA::NV - A2;
  constexpr int WB0 = TB ? 0 : B1, WB1 = TB ? 2 * LB::NS : B2 - B1, WB2 = TB ? 0 : LB::NV - B2;
  constexpr int LB0 = TB ? 0 : B1, LB1 = TB ? LB::NV : B2 - B1, LB2 = TB ? 0 : LB::NV - B2;
  const int nk = g.K / BK;
  auto iter = [&](auto setc, int kt) {
    constexpr int SET = decltype(setc)::value;
    const uint16_t* S = lds + (kt & 1) * STAGE;
    uint16_t* Sn = lds + ((kt + 1) & 1) * STAGE;
    const int kl = (kt + 1 + NSET) * BK;
    // step 0
    ldfrag(S, 1, 1);
    if constexpr (TA) { la.template store<SET, 0, LA::NS>(Sn); la.template load<SET, 0, LA::NV>(RA, kl); }
    else { la.template store<SET, 0, A1>(Sn); la.template load<SET, 0, A1>(RA, kl); }
    if constexpr (!TB) { lb.template store<SET, 0, B1>(Sn + BM * LDSK); lb.template load<SET, 0, B1>(RB, kl); }
    mfma_step(0);
    pipe_sched<MF, RD, WA0 + WB0, LA0 + LB0>();
    __builtin_amdgcn_sched_barrier(0);
    // step 1
    ldfrag(S, 2, 0);
    if constexpr (!TA) { la.template store<SET, A1, A2>(Sn); la.template load<SET, A1, A2>(RA, kl); }
    if constexpr (TB) { lb.template store<SET, 0, LB::NS>(Sn + BM * LDSK); lb.template load<SET, 0, LB::NV>(RB, kl); }
    else { lb.template store<SET, B1, B2>(Sn + BM * LDSK); lb.template load<SET, B1, B2>(RB, kl); }
    mfma_step(1);
    pipe_sched<MF, RD, WA1 + WB1, LA1 + LB1>();
    __builtin_amdgcn_sched_barrier(0);
    // step 2
    ldfrag(S, 3, 1);
    if constexpr (!TA) { la.template store<SET, A2, LA::NV>(Sn); la.template load<SET, A2, LA::NV>(RA, kl); }
    if constexpr (!TB) { lb.template store<SET, B2, LB::NV>(Sn + BM * LDSK); lb.template load<SET, B2, LB::NV>(RB, kl); }
    mfma_step(0);
    pipe_sched<MF, RD, WA2 + WB2, LA2 + LB2>();
    __builtin_amdgcn_sched_barrier(0);
    // every write of tile kt+1 and every read of tile kt is done past this barrier
    __syncthreads();
    // step 3, hiding the first fragment reads of tile kt+1
    ldfrag(Sn, 0, 0);
    mfma_step(1);
    pipe_sched<MF, RD, 0, 0>();
    __builtin_amdgcn_sched_barrier(0);
  };
  if constexpr (NSET == 2) {
    int kt = 0;
    for (; kt + 1 < nk; kt += 2) {
      iter(std::integral_constant<int, 1>(), kt);
      iter(std::integral_constant<int, 0>(), kt + 1);
    }
    if (kt < nk) iter(std::integral_constant<int, 1>(), kt);
  } else {
    for (int kt = 0; kt < nk; ++kt) iter(std::integral_constant<int, 0>(), kt);
  }
  __syncthreads();
  mfma_epilogue<BM, BN, WM, WN, EK>(g, acc, m0, n0, lds);
}

// --------------------------------------------- direct-to-LDS MFMA GEMM
// BM x BN workgroup tile (each 192 or 256), WM x WN waves (2 x 2; 2 x 4 for
// 256 x 256, where a second wave per SIMD keeps the MFMAs busy while the other
// wave stalls issuing its direct loads: 8% faster on that tile, while 4 x 2
// on 256 x 192 was slower than 2 x 2), 32-deep k tiles through 4 LDS stages,
// for K a multiple of 32.  Operands go from memory
// straight into LDS (buffer loads with the LDS bit: no register staging and no
// LDS write instructions), three k tiles ahead of the MFMAs.  LDS rows are
// unpadded and 16-byte chunks are XOR-swizzled by row so that both the 1 KB
// contiguous direct loads and the fragment reads are free of bank conflicts:
//   k-contiguous operand, tile [rows][32 k] (64 B rows):
//     chunk' = chunk ^ s(row), s = 2 row_1 ^ 3 row_2 ^ row_3 (row_i: bit i),
//     fragments are single 16-byte reads.  A 16-byte read is served in
//     groups of lanes such as {0-3, 32-35} (rows r..r+3, both halves of the
//     16-deep step); s keeps those groups, and groups of 8 or 16 consecutive
//     lanes, on distinct banks (SQ_LDS_BANK_CONFLICT reads 0; the earlier
//     s = (row_1 row_2) ^ (row_3 row_4) held only for consecutive lanes and
//     cost 1.6-1.9 conflict cycles per LDS instruction);
//   k-strided operand, tile [32 k][rows] (2 * rows bytes per k row):
//     chunk' = chunk ^ (((k & 3) << 1) | ((k & 1) << 3))  (256 rows),
//     chunk' = chunk ^ ((k & 3) << 1)                      (192 rows: the XOR
//     must stay inside aligned groups of 8 chunks),
//     fragments are two transposing 8-byte reads (ds_read_b64_tr_b16), each
//     of which hands lane i of a 16-lane group element (row e, column i) of
//     the 4 x 16 block the group fetched.
// The 192-wide tiles exist for the wave count: 256 CUs take 256x256 tiles of
// the block's products in 1.5 to 2.25 rounds, 256x192 or 192x192 tiles in
// whole rounds.  Ragged M / N edges rely on the buffer range check like the
// kernels above.
typedef short s16x4 __attribute__((ext_vector_type(4)));
#define JG_LDS(p) ((__attribute__((address_space(3))) void*)(p))
// First half of the workgroup barrier for the direct-loaded stages: this
// wave's LDS reads done (lgkmcnt 0) and at most NV of its direct loads still
// in flight (the loads of the two newest k tiles); s_barrier follows.  Unlike
// __syncthreads there is no release fence, which would wait for every direct
// load (they are LDS writes) and drain the prefetch; the empty asm statements
// keep the compiler from moving memory accesses across it.
template <int NV>
__device__ __forceinline__ void wait_vm_lds() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((NV & 15) | ((NV >> 4) << 14) | 0x70);  // vmcnt(NV) expcnt(7) lgkmcnt(0)
}

__device__ __forceinline__ int swz_n(int row) { return (((row >> 1) & 1) * 2) ^ (((row >> 2) & 1) * 3) ^ ((row >> 3) & 1); }
template <int ROWS>
__device__ __forceinline__ int swz_t(int k) {
  return ROWS == 256 ? (((k & 3) << 1) | ((k & 1) << 3)) : ((k & 3) << 1);
}

// One operand of the direct-to-LDS kernel: ROWS x 32 elements = ROWS * 64 B per
// k tile = NB direct loads of 1 KB, NL of them by each of the first NLW of the
// NW waves (the other waves load none of this operand); a wave's MFMAs read WR
// of the ROWS rows.
template <bool T, int ROWS, int NW, int WR>
struct DtlOp {
  static constexpr int NB = ROWS / 16;
  static constexpr int NL = (NB + NW - 1) / NW;
  static constexpr int NLW = NB / NL;
  static_assert(NB % NL == 0, "the loads of a k tile must split evenly over the loading waves");
  static constexpr int RB = ROWS * 2;   // bytes per k row (k-strided layout)
  static constexpr int CPR = ROWS / 8;  // chunks per k row
  static constexpr int FR = WR / 32;    // 32-row fragments per wave
  int voff[NL];  // per load: byte offset at k = 0
  int kmul;      // bytes per unit of k
  int fo[FR > 2 ? FR : 2];  // fragment read offsets (bytes)
  __device__ inline void init(int ld, int row0, int wrow0) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int t = 0; t < NL; ++t) {
      const int b = wave * NL + t;  // 1 KB block of the tile
      if (!T) {
        const int row = 16 * b + lane / 4, q = (lane % 4) ^ swz_n(row);
        voff[t] = ((row0 + row) * ld + 8 * q) * 2;
      } else {
        const int G = 64 * b + lane, kr = G / CPR, c = (G % CPR) ^ swz_t<ROWS>(kr);
        voff[t] = (kr * ld + row0 + 8 * c) * 2;
      }
    }
    kmul = T ? ld * 2 : 2;
    if (!T) {
      const int r = lane & 31;  // fragment row within a 32-row fragment
      fo[0] = (wrow0 + r) * 64 + (((lane >> 5)) ^ swz_n(r)) * 16;        // k16 step 0
      fo[1] = (wrow0 + r) * 64 + (((lane >> 5) + 2) ^ swz_n(r)) * 16;    // k16 step 1
    } else {
      const int g = (lane >> 4) & 3, i16 = lane & 15;
      const int kr = 8 * (g >> 1) + (i16 >> 2);  // row within the k16 step (first read)
#pragma unroll
      for (int i = 0; i < FR; ++i) {
        const int m = wrow0 + 32 * i + 16 * (g & 1) + 4 * (i16 & 3);
        fo[i] = kr * RB + (((m >> 3) ^ swz_t<ROWS>(kr)) << 4) + ((m >> 2) & 1) * 8;
      }
    }
  }
  // does this wave load any of the operand (wave-uniform)
  __device__ static inline bool loads(int wave) { return NLW == NW || wave < NLW; }
  // direct loads of the k tile at k0 into the stage at S (byte pointer)
  __device__ inline void load(__amdgpu_buffer_rsrc_t R, char* S, int k0) const {
    // wave-uniform: the LDS destination (M0) is then computed on the scalar unit
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (!loads(wave)) return;
#pragma unroll
    for (int t = 0; t < NL; ++t)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(R, JG_LDS(S + (wave * NL + t) * 1024), 16, voff[t] + k0 * kmul, 0, 0, 0);
  }
  // fragment i (32 rows) of k16 step kk from the stage at S
  __device__ inline bf16x8 frag(const char* S, int i, int kk) const {
    if (!T) {
      return __builtin_bit_cast(bf16x8, *(const u32x4*)(S + fo[kk] + i * 32 * 64));
    } else {
      const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) s16x4*)(S + fo[i] + kk * 16 * RB));
      const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) s16x4*)(S + fo[i] + kk * 16 * RB + 4 * RB));
      typedef short s16x8 __attribute__((ext_vector_type(8)));
      const s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      return __builtin_bit_cast(bf16x8, v);
    }
  }
};

// Epilogue of the direct-to-LDS kernel.  Each wave stages its accumulator
// tiles transposed in its own LDS region (one k stage per wave) and reads them
// back as 16 consecutive outputs of one row per lane; no workgroup barrier is
// needed because a wave reads back only what it wrote and one wave's LDS
// operations complete in issue order.  A tile that lies inside C takes the
// fast path: a whole row of FN accumulator tiles is staged at once and every
// global load its epilogue kind needs (old C, GELU input, bias) is issued
// before the first use, so the load latency is paid once per row of tiles
// instead of once per 32x32 tile.  Edge tiles take the checked path.
template <int BM, int BN, int WM, int WN, int EK>
__device__ __forceinline__ void dtl_epilogue(const GemmArgs& g, f32x16 (&acc)[BM / (32 * WM)][BN / (32 * WN)],
                                             int m0, int n0, float* T) {
  constexpr int FM = BM / (32 * WM), FN = BN / (32 * WN), ES = 36, TS = 32 * ES;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int h = lane >> 5, c32 = lane & 31;
  const int rr = lane & 31, cc = (lane >> 5) * 16;  // read-back: row rr, columns cc .. cc+15
  const int rbase = m0 + wm * (BM / WM), cbase = n0 + wn * (BN / WN);
  const bool vec_ok = (g.N % 8 == 0) && (g.epi.ldc % 8 == 0);
  const bool inner = vec_ok && m0 + BM <= g.M && n0 + BN <= g.N;
  const Epi& e = g.epi;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq)
        *(float4*)(T + j * TS + c32 * ES + 8 * gq + 4 * h) =
            make_float4(acc[i][j][4 * gq], acc[i][j][4 * gq + 1], acc[i][j][4 * gq + 2], acc[i][j][4 * gq + 3]);
    asm volatile("" ::: "memory");
    const int row = rbase + i * 32 + rr;
    if (inner) {
      float v[FN][2][8];
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int q = 0; q < 8; ++q) v[j][hf][q] = T[j * TS + (cc + 8 * hf + q) * ES + rr];
      asm volatile("" ::: "memory");
      // inputs of the epilogue kind, all in flight together
      u32x4 in0[FN][2], in1[FN][2];
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const int col = cbase + j * 32 + cc + 8 * hf;
          if constexpr (EK == EK_F32_ACC) {
            const u32x4* cp = (const u32x4*)((const float*)e.C + (size_t)row * e.ldc + col);
            in0[j][hf] = cp[0];
            in1[j][hf] = cp[1];
          } else if constexpr (EK == EK_BF16_ACC) {
            in0[j][hf] = *(const u32x4*)((const uint16_t*)e.C + (size_t)row * e.ldc + col);
          } else if constexpr (EK == EK_DGELU) {
            in0[j][hf] = *(const u32x4*)((const uint16_t*)e.aux + (size_t)row * e.ldaux + col);
          } else if constexpr (EK == EK_BIAS || EK == EK_GELU) {
            in0[j][hf] = *(const u32x4*)((const uint16_t*)e.bias + col);
          }
        }
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const int col = cbase + j * 32 + cc + 8 * hf;
          float* x = v[j][hf];
          if constexpr (EK == EK_F32 || EK == EK_F32_ACC) {
            if constexpr (EK == EK_F32_ACC) {
              const float4 o0 = __builtin_bit_cast(float4, in0[j][hf]), o1 = __builtin_bit_cast(float4, in1[j][hf]);
              x[0] += o0.x; x[1] += o0.y; x[2] += o0.z; x[3] += o0.w;
              x[4] += o1.x; x[5] += o1.y; x[6] += o1.z; x[7] += o1.w;
            }
            float4* cp = (float4*)((float*)e.C + (size_t)row * e.ldc + col);
            cp[0] = make_float4(x[0], x[1], x[2], x[3]);
            cp[1] = make_float4(x[4], x[5], x[6], x[7]);
          } else {
            float o[8];
            if constexpr (EK != EK_BF16) unpack8(in0[j][hf], o);
            if constexpr (EK == EK_BF16_ACC || EK == EK_BIAS || EK == EK_GELU) {
#pragma unroll
              for (int q = 0; q < 8; ++q) x[q] += o[q];
            }
            if constexpr (EK == EK_GELU) {
              *(u32x4*)((uint16_t*)e.aux + (size_t)row * e.ldaux + col) = pack8(x);
#pragma unroll
              for (int q = 0; q < 8; ++q) x[q] = gelu_tanh(x[q]);
            }
            if constexpr (EK == EK_DGELU) {
#pragma unroll
              for (int q = 0; q < 8; ++q) x[q] *= gelu_tanh_grad(o[q]);
            }
            *(u32x4*)((uint16_t*)e.C + (size_t)row * e.ldc + col) = pack8(x);
          }
        }
    } else {
#pragma unroll 1
      for (int j = 0; j < FN; ++j)
#pragma unroll 1
        for (int hf = 0; hf < 2; ++hf) {
          const int col = cbase + j * 32 + cc + 8 * hf;
          if (row >= g.M) continue;
          float v[8];
#pragma unroll
          for (int q = 0; q < 8; ++q) v[q] = T[j * TS + (cc + 8 * hf + q) * ES + rr];
          if (vec_ok && col + 8 <= g.N) {
            epi8<EK>(e, row, col, v);
          } else {
#pragma unroll 1
            for (int q = 0; q < 8; ++q)
              if (col + q < g.N) epi1<EK>(e, row, col + q, v[q]);
          }
        }
    }
    // the next row's staging writes must not move above this row's reads
    asm volatile("" ::: "memory");
  }
}

template <bool TA, bool TB, int EK, int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(64 * WM * WN) void gemm_dtl_kernel(GemmGroup gg) {
  constexpr int BK = 32, NW = WM * WN, FM = BM / (32 * WM), FN = BN / (32 * WN);
  constexpr int SB = BM * 64;  // byte offset of the B tile in a stage
  constexpr int STG = 32768;   // bytes per stage (room for 256 + 256 rows)
  // one variable per stage: every LDS access names its stage statically, so
  // the compiler can tell the fragment reads of one stage from the direct
  // loads still landing in another and does not wait for the latter
  __shared__ __attribute__((aligned(1024))) char st0[STG];
  __shared__ __attribute__((aligned(1024))) char st1[STG];
  __shared__ __attribute__((aligned(1024))) char st2[STG];
  __shared__ __attribute__((aligned(1024))) char st3[STG];

  // the first tiles0 workgroups compute problem 0, the rest problem 1
  const int sel = (int)blockIdx.x >= gg.tiles0 ? 1 : 0;
  const GemmArgs& g = gg.p[sel];
  const int local = (int)blockIdx.x - sel * gg.tiles0;
  const int tiles_m = (g.M + BM - 1) / BM, tiles_n = (g.N + BN - 1) / BN;
  int tm, tn;
  tile_coords(xcd_remap(local, tiles_m * tiles_n), tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;

  typedef DtlOp<TA, BM, NW, BM / WM> OpA;
  typedef DtlOp<TB, BN, NW, BN / WN> OpB;
  OpA oa;
  OpB ob;
  oa.init(g.lda, m0, wm * (BM / WM));
  ob.init(g.ldb, n0, wn * (BN / WN));
  const long ext_a = TA ? ((long)(g.K - 1) * g.lda + g.M) * 2 : ((long)(g.M - 1) * g.lda + g.K) * 2;
  const long ext_b = TB ? ((long)(g.K - 1) * g.ldb + g.N) * 2 : ((long)(g.N - 1) * g.ldb + g.K) * 2;
  const __amdgpu_buffer_rsrc_t RA = make_rsrc(g.A, ext_a), RB = make_rsrc(g.B, ext_b);

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  auto stage = [&](auto ic) -> char* {
    constexpr int c = decltype(ic)::value & 3;
    if constexpr (c == 0) return st0;
    else if constexpr (c == 1) return st1;
    else if constexpr (c == 2) return st2;
    else return st3;
  };
  bf16x8 fa[2][FM], fb[2][FN];
  auto ldfrag = [&](const char* S, int kk, int buf) {
#pragma unroll
    for (int i = 0; i < FM; ++i) fa[buf][i] = oa.frag(S, i, kk);
#pragma unroll
    for (int j = 0; j < FN; ++j) fb[buf][j] = ob.frag(S + SB, j, kk);
  };
  auto mfma_step = [&](int buf) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[buf][i], fb[buf][j], acc[i][j], 0, 0, 0);
  };
  auto load_tile = [&](char* S, int t) {
    oa.load(RA, S, t * BK);
    ob.load(RB, S + SB, t * BK);
  };

  // prologue: tiles 0, 1, 2 in flight; wait for tile 0
  constexpr int NL = OpA::NL + OpB::NL;  // direct loads per (fully loading) wave per k tile
  // Wait until at most two k tiles of this wave's own direct loads are in
  // flight, then meet the other waves: the waves that load only one operand
  // (or none) wait for fewer.
  const bool lda_w = OpA::loads(wave), ldb_w = OpB::loads(wave);
  auto tile_barrier = [&]() {
    if (lda_w && ldb_w) wait_vm_lds<2 * NL>();
    else if (lda_w) wait_vm_lds<2 * OpA::NL>();
    else if (ldb_w) wait_vm_lds<2 * OpB::NL>();
    else wait_vm_lds<0>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };
  const int nk = g.K / BK;
  // Every wave loads both operands: A's loads of a k tile go with the first
  // MFMA step, B's with the second.  A wave stalls while the memory pipeline
  // cannot take its next direct load, and with one wave per SIMD the MFMAs
  // stall with it; spread over both steps, the loads cost 3-4% less time in
  // the weight-gradient products.
  constexpr bool SPLIT = OpA::NLW == NW && OpB::NLW == NW;
  load_tile(st0, 0);
  load_tile(st1, 1);
  load_tile(st2, 2);
  tile_barrier();  // tiles 1 and 2 may still fly
  ldfrag(st0, 0, 0);

  constexpr int RD = (TA ? 2 : 1) * FM + (TB ? 2 : 1) * FN;  // LDS reads per k16 step
  // k tile kt is read from stage kt % 4, tile kt+3 loads into stage (kt+3) % 4
  auto iter = [&](auto ic, int kt) {
    constexpr int c = decltype(ic)::value;
    const char* S = stage(std::integral_constant<int, c>());
    const char* Sn = stage(std::integral_constant<int, c + 1>());
    // step 0: fragments of step 1 and the direct loads of tile kt+3 (its stage
    // was last read before the previous barrier): all of them, or with SPLIT
    // only A's, B's following in step 1
    ldfrag(S, 1, 1);
    char* Sx = stage(std::integral_constant<int, c + 3>());
    if constexpr (SPLIT) oa.load(RA, Sx, (kt + 3) * BK);
    else load_tile(Sx, kt + 3);
    mfma_step(0);
    pipe_sched<FM * FN, RD, 0, SPLIT ? OpA::NL : NL>();
    __builtin_amdgcn_sched_barrier(0);
    // tile kt+1 has landed once at most the loads of tile kt+2 and those of
    // tile kt+3 issued so far fly
    if constexpr (SPLIT) {
      wait_vm_lds<NL + OpA::NL>();
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
    } else {
      tile_barrier();
    }
    // step 1, hiding the first fragment reads of tile kt+1
    ldfrag(Sn, 0, 0);
    if constexpr (SPLIT) ob.load(RB, Sx + SB, (kt + 3) * BK);
    mfma_step(1);
    pipe_sched<FM * FN, RD, 0, SPLIT ? OpB::NL : 0>();
    __builtin_amdgcn_sched_barrier(0);
  };
  int kt = 0;
  for (; kt + 3 < nk; kt += 4) {
    iter(std::integral_constant<int, 0>(), kt);
    iter(std::integral_constant<int, 1>(), kt + 1);
    iter(std::integral_constant<int, 2>(), kt + 2);
    iter(std::integral_constant<int, 3>(), kt + 3);
  }
  if (kt < nk) iter(std::integral_constant<int, 0>(), kt);
  if (kt + 1 < nk) iter(std::integral_constant<int, 1>(), kt + 1);
  if (kt + 2 < nk) iter(std::integral_constant<int, 2>(), kt + 2);
  // every direct load has landed and every wave is past its last fragment
  // read before the stages are reused as per-wave epilogue staging
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  // per-wave staging: FN 32 x 36 fp32 tiles (at most 18 KB), NW / 4 waves per stage
  constexpr int TQ = NW / 4, TB_ = STG / TQ;
  static_assert(FN * 32 * 36 * 4 <= TB_, "epilogue staging exceeds its share of a stage");
  const int ws = wave / TQ;
  float* T = (float*)((ws == 0 ? st0 : ws == 1 ? st1 : ws == 2 ? st2 : st3) + (wave % TQ) * TB_);
  dtl_epilogue<BM, BN, WM, WN, EK>(g, acc, m0, n0, T);
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
static GemmGroup single(const GemmArgs& g) {
  GemmGroup r;
  r.p[0] = g;
  r.np = 1;
  return r;
}

// Sets a kernel's dynamic-LDS limit once per device (bit d of `bits`; safe to
// race, the call is idempotent).
static int reserve_lds(std::atomic<unsigned long long>& bits, const void* kern, size_t lds, const char* who) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev > 63) {
    set_error(std::string(who) + ": no current device");
    return 3;
  }
  if (!(bits.load(std::memory_order_acquire) & (1ull << dev))) {
    if (hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess) {
      set_error(std::string(who) + ": cannot reserve the LDS tile stages");
      return 3;
    }
    bits.fetch_or(1ull << dev, std::memory_order_acq_rel);
  }
  return 0;
}

template <int BM, int BN, int BK, int WM, int WN, bool TA, bool TB, int EK>
static int launch_pipe(const GemmGroup& gr, hipStream_t s) {
  GemmGroup g = gr;
  int tiles = 0;
  for (int p = 0; p < g.np; ++p) {
    const int t = ((g.p[p].M + BM - 1) / BM) * ((g.p[p].N + BN - 1) / BN);
    if (p == 0) g.tiles0 = t;
    tiles += t;
  }
  if (g.np == 1) g.tiles0 = tiles;
  const size_t lds = 2 * (size_t)(BM + BN) * (BK + 8) * sizeof(uint16_t);
  void (*kern)(GemmGroup) = gemm_pipe_kernel<BM, BN, BK, WM, WN, TA, TB, EK>;
  static std::atomic<unsigned long long> attr{0};
  if (int rc = reserve_lds(attr, (const void*)kern, lds, "gemm_pipe")) return rc;
  launch(kern, dim3(tiles), dim3(WM * WN * 64), (uint32_t)lds, s, g);
  JG_CHECK_LAUNCH("gemm_pipe");
  return 0;
}

template <int BM, int BN, int BK, int WM, int WN, bool TA, bool TB, int EK, bool PIPE>
static int launch_mfma(const GemmArgs& g, hipStream_t s) {
  if constexpr (PIPE) {
    return launch_pipe<BM, BN, BK, WM, WN, TA, TB, EK>(single(g), s);
  } else {
    const int tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
    const size_t lds = 2 * (size_t)(BM + BN) * (BK + 8) * sizeof(uint16_t);
    void (*kern)(GemmArgs) = gemm_mfma_kernel<BM, BN, BK, WM, WN, TA, TB, EK>;
    static std::atomic<unsigned long long> attr{0};
    if (int rc = reserve_lds(attr, (const void*)kern, lds, "gemm_mfma")) return rc;
    launch(kern, dim3(tiles), dim3(WM * WN * 64), (uint32_t)lds, s, g);
    JG_CHECK_LAUNCH("gemm_mfma");
    return 0;
  }
}

template <bool TA, bool TB, int EK, int BM, int BN, int WM = 2, int WN = 2>
static int launch_dtl(const GemmGroup& gr, hipStream_t s) {
  GemmGroup g = gr;
  int tiles = 0;
  for (int p = 0; p < g.np; ++p) {
    const int t = ((g.p[p].M + BM - 1) / BM) * ((g.p[p].N + BN - 1) / BN);
    if (p == 0) g.tiles0 = t;
    tiles += t;
  }
  if (g.np == 1) g.tiles0 = tiles;
  launch(gemm_dtl_kernel<TA, TB, EK, BM, BN, WM, WN>, dim3(tiles), dim3(64 * WM * WN), 0u, s, g);
  JG_CHECK_LAUNCH("gemm_dtl");
  return 0;
}

// Tile shape of the direct-to-LDS kernel: the one with the least estimated
// time = rounds of 256 workgroups x tile area / relative tile efficiency
// (smaller tiles re-read more operand bytes per MFMA).  0: 256x256 (8 waves),
// 1: 256x192, 2: 192x256, 3: 192x192.  Rounds count whole rounds of problem
// 0's tiles; the tiles of a second problem with a shorter contraction are
// shorter and fill in behind them (the dispatcher hands a freed CU the next
// workgroup), so they add their share of a round; equal contractions share
// whole rounds.
static int dtl_shape(const GemmGroup& g) {
  static const int bm[4] = {256, 256, 192, 192}, bn[4] = {256, 192, 256, 192};
  static const double eff[4] = {1.0, 0.95, 0.95, 0.9};
  int best = 0;
  double bt = 1e300;
  for (int i = 0; i < 4; ++i) {
    long tl[2] = {0, 0};
    for (int p = 0; p < g.np; ++p)
      tl[p] = (long)((g.p[p].M + bm[i] - 1) / bm[i]) * ((g.p[p].N + bn[i] - 1) / bn[i]);
    double rounds;
    if (g.np == 1 || g.p[1].K == g.p[0].K) {
      rounds = (double)((tl[0] + tl[1] + 255) / 256);
    } else {
      const double work = tl[0] + (double)tl[1] * g.p[1].K / g.p[0].K;
      rounds = std::max((double)((tl[0] + 255) / 256), work / 256.0);
    }
    const double t = rounds * bm[i] * bn[i] / eff[i];
    if (t < bt * 0.999) { bt = t; best = i; }
  }
  return best;
}

// The direct-to-LDS kernel serves the products with a k-strided B operand
// (input and weight gradients); -1 for the others.
template <bool TA, bool TB, int EK>
struct DtlLaunch {
  static int run(const GemmGroup& g, hipStream_t s, int shape) {
    switch (shape) {
      case 1: return launch_dtl<TA, TB, EK, 256, 192>(g, s);
      case 2: return launch_dtl<TA, TB, EK, 192, 256>(g, s);
      case 3: return launch_dtl<TA, TB, EK, 192, 192>(g, s);
      default: return launch_dtl<TA, TB, EK, 256, 256, 2, 4>(g, s);
    }
  }
};
template <bool TA, int EK>
struct DtlLaunch<TA, false, EK> {
  static int run(const GemmGroup&, hipStream_t, int) { return -1; }
};

// The direct-to-LDS kernel computes 32-bit byte offsets up to three k tiles
// past K; they must stay below 2^31.
static bool dtl_fits(const GemmArgs& g) {
  const double kx = (double)g.K + 128.0;
  const double ea = 2.0 * (g.ta ? kx * g.lda + g.M : (double)g.M * g.lda + kx);
  const double eb = 2.0 * (g.tb ? kx * g.ldb + g.N : (double)g.N * g.ldb + kx);
  return g.K % 32 == 0 && ea < 2147483000.0 && eb < 2147483000.0;
}

template <bool TA, bool TB, int EK>
static int launch_cfg(const GemmArgs& g, hipStream_t s, int cfg) {
  if (TB && cfg >= 8 && cfg <= 12 && dtl_fits(g)) {
    const GemmGroup one = single(g);
    const int rc = DtlLaunch<TA, TB, EK>::run(one, s, cfg == 8 ? dtl_shape(one) : cfg - 9);
    if (rc >= 0) return rc;
  }
  // K not a multiple of the 64-deep k tile: the edge-checked kernel
  if (g.K % 64 != 0) return launch_mfma<128, 128, 64, 2, 2, TA, TB, EK, false>(g, s);
  switch (cfg) {
    case 1: return launch_mfma<128, 128, 64, 2, 2, TA, TB, EK, true>(g, s);
    case 2: return launch_mfma<256, 128, 64, 2, 2, TA, TB, EK, true>(g, s);
    case 6: return launch_mfma<256, 256, 64, 2, 4, TA, TB, EK, true>(g, s);
    default: return launch_mfma<256, 256, 64, 2, 2, TA, TB, EK, true>(g, s);
  }
}

template <bool TA, bool TB>
static int launch_kind(const GemmArgs& g, hipStream_t s, int cfg, int ek) {
  switch (ek) {
    case EK_F32: return launch_cfg<TA, TB, EK_F32>(g, s, cfg);
    case EK_F32_ACC: return launch_cfg<TA, TB, EK_F32_ACC>(g, s, cfg);
    case EK_BF16: return launch_cfg<TA, TB, EK_BF16>(g, s, cfg);
    case EK_BF16_ACC: return launch_cfg<TA, TB, EK_BF16_ACC>(g, s, cfg);
    case EK_BIAS: return launch_cfg<TA, TB, EK_BIAS>(g, s, cfg);
    case EK_GELU: return launch_cfg<TA, TB, EK_GELU>(g, s, cfg);
    default: return launch_cfg<TA, TB, EK_DGELU>(g, s, cfg);
  }
}

// The output kind of an epilogue, or -1 if the MFMA epilogues do not cover it.
static int epi_kind(const Epi& e) {
  const bool bias = e.bias != nullptr;
  if (bias && e.bias_dt != BF16) return -1;
  if ((e.mode == EPI_GELU_FWD || e.mode == EPI_GELU_BWD) && e.aux_dt != BF16) return -1;
  if (e.mode == EPI_STORE && !bias) {
    if (e.beta != 0.f && e.beta != 1.f) return -1;
    if (e.c_dt == F32) return e.beta != 0.f ? EK_F32_ACC : EK_F32;
    return e.beta != 0.f ? EK_BF16_ACC : EK_BF16;
  }
  if (e.beta != 0.f || e.c_dt != BF16) return -1;
  if (e.mode == EPI_STORE) return EK_BIAS;
  if (e.mode == EPI_GELU_FWD) return bias ? EK_GELU : -1;
  return bias ? -1 : EK_DGELU;
}

static int prof_class(const GemmArgs& g) {
  if (!g.ta && !g.tb) return PROF_GEMM_FWD;
  if (!g.ta && g.tb) return PROF_GEMM_DGRAD;
  if (g.ta && g.tb) return PROF_GEMM_WGRAD;
  return PROF_NONE;
}

static int gemm_launch(const GemmArgs& g, hipStream_t s);

int gemm(const GemmArgs& g, hipStream_t s) {
  const int pi = prof_begin(prof_class(g));
  const int rc = gemm_launch(g, s);
  prof_end(pi, 2.0 * g.M * g.N * (double)g.K);
  return rc;
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// The epilogue kind of g if the MFMA kernels can compute it (bf16 operands,
// 16-byte aligned rows, 32-bit operand extents), else -1.
static int mfma_kind(const GemmArgs& g) {
  bool mfma = g.a_dt == BF16 && g.b_dt == BF16 && g.K > 0 && aligned16(g.A) && aligned16(g.B) &&
              g.lda % 8 == 0 && g.ldb % 8 == 0;
  if (mfma) mfma = (g.ta ? g.M % 8 == 0 : g.K % 8 == 0) && (g.tb ? g.N % 8 == 0 : g.K % 8 == 0);
  const int ek = mfma ? epi_kind(g.epi) : -1;
  if (ek >= 0 && (g.epi.ldc % 8 != 0 || !aligned16(g.epi.C) || (g.epi.aux && (g.epi.ldaux % 8 || !aligned16(g.epi.aux)))))
    return -1;
  // operand extents must fit a 32-bit buffer offset
  const double ea = 2.0 * (g.ta ? (double)g.K * g.lda : (double)g.M * g.lda);
  const double eb = 2.0 * (g.tb ? (double)g.K * g.ldb : (double)g.N * g.ldb);
  if (ea >= 2147483000.0 || eb >= 2147483000.0) return -1;
  return ek;
}

static int gemm_launch(const GemmArgs& g, hipStream_t s) {
  if (g.M < 0 || g.N < 0 || g.K < 0 || !g.A || !g.B || !g.epi.C) {
    set_error("gemm: invalid arguments");
    return 1;
  }
  if (g.M == 0 || g.N == 0) return 0;
  const int ek = mfma_kind(g);
  if (ek >= 0) {
    // default: products with a k-strided B operand (weight and input
    // gradients) take the direct-to-LDS kernel with the tile shape that best
    // fills whole rounds of 256 CUs; the forward product takes the 8-wave
    // register-staged 256x256 kernel, or 128x128 for grids too small to
    // cover a quarter of the chip
    const long t256 = (long)((g.M + 255) / 256) * ((g.N + 255) / 256);
    int cfg;
    if (g.tb && dtl_fits(g)) cfg = 8;
    else if (t256 < 64) cfg = 1;
    else if (!g.ta && !g.tb) cfg = 6;
    else cfg = 4;
    if (!g.ta && !g.tb) return launch_kind<false, false>(g, s, cfg, ek);
    if (!g.ta && g.tb) return launch_kind<false, true>(g, s, cfg, ek);
    if (g.ta && g.tb) return launch_kind<true, true>(g, s, cfg, ek);
    return launch_kind<true, false>(g, s, cfg, ek);
  }
  // the VALU kernel also covers an empty contraction (K = 0): it still
  // applies the epilogue (bias, beta)
  dim3 grid((g.N + 63) / 64, (g.M + 63) / 64);
  launch(gemm_valu_kernel, grid, dim3(256), 0u, s, g);
  JG_CHECK_LAUNCH("gemm_valu");
  return 0;
}

template <bool TA, int EK>
static int launch_group(const GemmGroup& g, hipStream_t s) {
  return DtlLaunch<TA, true, EK>::run(g, s, dtl_shape(g));
}

template <int EK>
static int launch_fwd_group(const GemmGroup& g, hipStream_t s) {
  long t256 = 0;
  for (int p = 0; p < g.np; ++p) t256 += (long)((g.p[p].M + 255) / 256) * ((g.p[p].N + 255) / 256);
  if (t256 < 64) return launch_pipe<128, 128, 64, 2, 2, false, false, EK>(g, s);
  return launch_pipe<256, 256, 64, 2, 4, false, false, EK>(g, s);
}

int gemm2(const GemmArgs& a, const GemmArgs& b, hipStream_t s) {
  // one grouped launch when both products take the same kernel: the
  // direct-to-LDS kernel (k-strided B: input and weight gradients) or the
  // register-staged one (forward products, K a multiple of its 64-deep tile)
  const int ek = (a.M > 0 && a.N > 0 && b.M > 0 && b.N > 0 && a.A && a.B && a.epi.C && b.A && b.B && b.epi.C)
                     ? mfma_kind(a) : -1;
  const bool same = ek >= 0 && mfma_kind(b) == ek && a.ta == b.ta && a.tb == b.tb;
  const bool fwd = same && !a.ta && !a.tb && a.K % 64 == 0 && b.K % 64 == 0;
  const bool grouped = fwd || (same && a.tb && dtl_fits(a) && dtl_fits(b));
  if (!grouped) {
    int rc = gemm(a, s);
    return rc ? rc : gemm(b, s);
  }
  // the longer contraction first: its tiles take the whole rounds, the other's fill in
  GemmGroup g;
  g.np = 2;
  g.p[0] = b.K > a.K ? b : a;
  g.p[1] = b.K > a.K ? a : b;
  const int pi = prof_begin(prof_class(a));
  int rc;
  if (fwd) {
    switch (ek) {
#define JG_FWD(E) case E: rc = launch_fwd_group<E>(g, s); break;
      JG_FWD(EK_F32) JG_FWD(EK_F32_ACC) JG_FWD(EK_BF16) JG_FWD(EK_BF16_ACC) JG_FWD(EK_BIAS) JG_FWD(EK_GELU)
      default: rc = launch_fwd_group<EK_DGELU>(g, s); break;
#undef JG_FWD
    }
    prof_end(pi, 2.0 * ((double)a.M * a.N * a.K + (double)b.M * b.N * b.K));
    return rc;
  }
  switch (ek) {
#define JG_GRP(E) case E: rc = a.ta ? launch_group<true, E>(g, s) : launch_group<false, E>(g, s); break;
    JG_GRP(EK_F32) JG_GRP(EK_F32_ACC) JG_GRP(EK_BF16) JG_GRP(EK_BF16_ACC) JG_GRP(EK_BIAS) JG_GRP(EK_GELU)
    default: rc = a.ta ? launch_group<true, EK_DGELU>(g, s) : launch_group<false, EK_DGELU>(g, s); break;
#undef JG_GRP
  }
  prof_end(pi, 2.0 * ((double)a.M * a.N * a.K + (double)b.M * b.N * b.K));
  return rc;
}

// Explicit instantiations of the direct-to-LDS kernels the dispatch can reach
// (the host-side launch stubs of kernel templates reached only through the
// shape switch are otherwise not always emitted).
#define JG_DTL_SHAPES(TA, EK)                                            \
  template __global__ void gemm_dtl_kernel<TA, true, EK, 256, 256, 2, 4>(GemmGroup); \
  template __global__ void gemm_dtl_kernel<TA, true, EK, 256, 192, 2, 2>(GemmGroup); \
  template __global__ void gemm_dtl_kernel<TA, true, EK, 192, 256, 2, 2>(GemmGroup); \
  template __global__ void gemm_dtl_kernel<TA, true, EK, 192, 192, 2, 2>(GemmGroup);
#define JG_DTL_KINDS(TA) \
  JG_DTL_SHAPES(TA, 0) JG_DTL_SHAPES(TA, 1) JG_DTL_SHAPES(TA, 2) JG_DTL_SHAPES(TA, 3) JG_DTL_SHAPES(TA, 4) \
  JG_DTL_SHAPES(TA, 5) JG_DTL_SHAPES(TA, 6)
JG_DTL_KINDS(false)
JG_DTL_KINDS(true)
#undef JG_DTL_KINDS
#undef JG_DTL_SHAPES

}  // namespace jg

