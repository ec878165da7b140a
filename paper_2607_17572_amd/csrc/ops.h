// Memory-bound kernels of the DiT forward/backward and the JAGG steps.
#pragma once
#include "common.h"

namespace jg {

// Token rows are stored stream-major: the text rows of all B samples first
// (sample b's text rows at b*nt .. b*nt+nt-1), then the image rows
// (sample b's image rows at B*nt + b*ni ...).  Every per-stream GEMM thus
// sees one contiguous row range, and a single-stream block sees all rows.
struct RowMap {
  int B, nt, ni;
  __host__ __device__ int rows_txt() const { return B * nt; }
  __host__ __device__ int rows() const { return B * (nt + ni); }
};

// Row chunks for deterministic column reductions: chunks never straddle a
// sample or a stream.  R rows per chunk.
struct Chunks {
  int B, nt, ni, R;
  __host__ __device__ int ct() const { return (nt + R - 1) / R; }
  __host__ __device__ int ci() const { return (ni + R - 1) / R; }
  __host__ __device__ int count() const { return B * (ct() + ci()); }
};

constexpr int RED_ROWS = 32;  // rows per reduction chunk
// rows per block of the LayerNorm/adaLN backward, whose partial sums are per
// block: the pair's 9216 rows make 1152 blocks, which the CUs take up as they
// free (whole 32-row chunks left 32 of 256 CUs with two blocks, the rest with one)
constexpr int LN_ROWS = 8;

// ---- small-M linear layers (time MLP, adaLN modulation): M = batch <= 64 ----
// out[b][j] = sum_d act(in[b][d]) W[j][d] + bias[j];  act: 0 identity, 1 SiLU.
int small_linear_fwd(const float* in, int act, int B, int Din, const void* W, const void* bias, int w_dt,
                     float* out, int Dout, hipStream_t s);
// dW[j][d] (+)= sum_b dout[b][j] act(in[b][d]) ; db[j] (+)= sum_b dout[b][j];
// din[b][d] (+)= sum_j dout[b][j] W[j][d]  (fp32, overwritten, or added to
// when din_acc; nullptr to skip).
// `part` is workspace of small_linear_bwd_part_floats() floats.
size_t small_linear_bwd_part_floats(int B, int Din, int Dout);
int small_linear_bwd(const float* dout, const float* in, int act, int B, int Din, const void* W, int w_dt,
                     int Dout, void* dW, void* db, int g_dt, float beta, float* din, float* part,
                     hipStream_t s, bool din_acc = false);

// ---- time embedding: temb[b][k] = cos(1000 t_b w_k), temb[b][F/2+k] = sin(...) ----
struct TVals { float t[64]; };
int time_embed(const TVals& tv, int B, int F, float* temb, hipStream_t s);

// elementwise y = f(x) on fp32 arrays: op 0 silu, 1 silu_grad-multiply (y = y * silu'(x))
int silu_fwd(const float* x, float* y, size_t n, hipStream_t s);
int mul_silu_grad(float* y, const float* x, size_t n, hipStream_t s);

// ---- LayerNorm (no affine) + adaLN modulate ----
// a = LN(x) * (1 + scale[b]) + shift[b]; rows [row0, row0 + nrows) of the map.
// mod_txt / mod_img: fp32 [B][mod_w]; shift at column sh_off, scale at sc_off.
int ln_mod_fwd(const void* x, int act_dt, int D, RowMap rm, int row0, int nrows, const float* mod_txt,
               const float* mod_img, int mod_w, int sh_off, int sc_off, void* a, float* mean, float* rstd,
               hipStream_t s);
// g[r] = g_in[r] + LN_bwd(dA * (1 + scale)) and partials of sum dA*xhat
// (-> part_scale) and sum dA (-> part_shift) per chunk of LN_ROWS rows,
// [chunk][D].  g_in is fp32 (it may be g itself) or, with bf16 activations, bf16.
int ln_mod_bwd(const float* dA, const void* x, int act_dt, int D, RowMap rm, int row0, int nrows,
               const float* mean, const float* rstd, const float* mod_txt, const float* mod_img, int mod_w,
               int sc_off, const void* g_in, int g_in_dt, float* g, float* part_scale, float* part_shift,
               hipStream_t s);

// ---- gated residual ----
// xo = xi + gate[b] * y  (rows [row0, row0+nrows))
int gated_residual(const void* xi, const void* y, int act_dt, int D, int ld_y, RowMap rm, int row0, int nrows,
                   const float* mod_txt, const float* mod_img, int mod_w, int gate_off, void* xo,
                   hipStream_t s);
// dY = g * gate[b] (act dtype), partials: part_gate = sum g*y, part_bias = sum dY.
// g is fp32 or, with bf16 activations, bf16 (g_dt).
int gate_bwd(const void* g, int g_dt, const void* y, int act_dt, int D, RowMap rm, int row0, int nrows,
             const float* mod_txt, const float* mod_img, int mod_w, int gate_off, void* dY, int ld_dy,
             float* part_gate, float* part_bias, hipStream_t s);

// ---- q/k RMSNorm + 2-D rotary embedding ----
struct Rope {
  int H, Dh, nt, ni, gw;  // image tokens on a grid of width gw
};
// proj: [rows][ld] with q at col 0, k at D, v at 2D (raw).  Writes head-major
// Qh/Kh/Vh [B][H][N][Dh] (act dtype), rinv_q/rinv_k [rows][H].
// Gains are per stream (text rows use g[0], image rows g[1]); pass the same
// pointers twice for a single-stream block.
struct Gains { const void* q[2]; const void* k[2]; };
int qk_norm_rope_fwd(const void* proj, int ld, int act_dt, RowMap rm, Rope rp, Gains gn,
                     void* Qh, void* Kh, void* Vh, float* rinv_q, float* rinv_k, hipStream_t s);
// dQh/dKh/dVh head-major (dt_d) -> dproj[row][0..3D) (act dtype, ld), dgain partials
// [chunk * QK_PARTS + sub][2*Dh] (QK_PARTS sub-chunks per reduction chunk).
constexpr int QK_PARTS = 4;
int qk_norm_rope_bwd(const void* dQh, const void* dKh, const void* dVh, int dt_d, const void* proj, int ld,
                     int act_dt, RowMap rm, Rope rp, Gains gn, const float* rinv_q,
                     const float* rinv_k, void* dproj, int ld_d, float* part_gain, hipStream_t s);

// ---- reductions ----
// column sums of X[rows][ld] (dtype) over chunks -> part[chunk][N]
int colsum_partials(const void* X, int dt, int ld, int N, RowMap rm, int row0, int nrows, float* part,
                    hipStream_t s);
// Per-sample reduction: out[b*out_stride + out_off + c] = sum over chunks of sample b (of the
// chunks belonging to rows [row0, row0+nrows)) of part[chunk][c].  Overwrites.
// R: rows per chunk of the partials.
int reduce_per_sample(const float* part, int N, RowMap rm, int row0, int nrows, float* out, int out_stride,
                      int out_off, hipStream_t s, int R = RED_ROWS);
// Whole reduction into a parameter gradient: g[c] = beta*g[c] + sum_chunks part[chunk*ld + c].
int reduce_to_grad(const float* part, int ld, int chunk0, int nchunk, int N, void* g, int g_dt,
                   float beta, hipStream_t s);
int chunk_range(RowMap rm, int row0, int nrows, int* c0, int* nc, int R = RED_ROWS);

// A list of independent chunk reductions run as one launch, each job with the
// arithmetic (and so the bits) of reduce_per_sample or reduce_to_grad.
struct RedJob {
  const float* part = nullptr;
  int ld = 0, N = 0;          // partial row stride and columns
  int kind = 0;               // 0: per sample, 1: into a parameter gradient
  Chunks ch{};                // per sample: chunk geometry
  int c0 = 0, nc = 0;         // chunk range
  float* out = nullptr;       // per sample: out[b*out_stride + out_off + c]
  int out_stride = 0, out_off = 0;
  void* g = nullptr;          // gradient: g[c] = beta*g[c] + sum
  int g_dt = 0;
  float beta = 0.f;
  int blk0 = 0;               // first block of the job (set by reduce_jobs)
};
constexpr int RED_MAX_JOBS = 8;
RedJob per_sample_job(const float* part, int N, RowMap rm, int row0, int nrows, float* out, int out_stride,
                      int out_off, int R = RED_ROWS);
RedJob to_grad_job(const float* part, int ld, int chunk0, int nchunk, int N, void* g, int g_dt, float beta);
// Runs jobs[0..n) (n <= RED_MAX_JOBS) in one launch; 1 on an invalid job.
int reduce_jobs(const RedJob* jobs, int n, hipStream_t s);

// ---- misc ----
int patchify(const void* z, int dt, int B, int C, int Hh, int Ww, int p, void* out, hipStream_t s);
int unpatchify(const void* x, int dt, int B, int C, int Hh, int Ww, int p, void* z, hipStream_t s);
int convert(const void* x, int dt_in, void* y, int dt_out, size_t n, hipStream_t s);
int fill_zero(void* x, size_t bytes, hipStream_t s);

// ---- JAGG aggregation (Eq. s_base / s_corr) ----
struct AggArgs {
  const void* s[64];
  float wb[64], wc[64];  // (1 - alpha_j), alpha_j
  int W;
  size_t n;              // elements per s_j
  size_t split;          // elements [0, split) -> dst*0, [split, n) -> dst*1 at (e - split)
  void* base0; void* base1; void* corr0; void* corr1;
  int in_dt, out_dt;
};
int aggregate(const AggArgs& a, hipStream_t s);

// ---- group scores: mean pairwise cosine of W vectors of n elements (fp64) ----
struct ScoreArgs {
  const void* h[16];
  int W;
  size_t n;
  int dt;
};
size_t score_part_doubles(int W);
int group_scores(const ScoreArgs& a, double* part, double* score_dev, hipStream_t s);

// ---- GRPO upstream gradients (Phase 2) and their composites (Phase 3) ----
// Rollout data of one window in the batch-B output layout: element e belongs
// to sample e / len0 when e < split, else to sample (e - split) / len1.
constexpr int GRPO_MAX_W = 16;
struct GrpoArgs {
  const void* v[GRPO_MAX_W];      // model outputs v_j
  int vb[GRPO_MAX_W], vk[GRPO_MAX_W];  // v_j: samples vk .. vk+B-1 of a batch-vb array
  const void* z[GRPO_MAX_W + 1];  // latents z_0 .. z_W
  int W, B, dt;
  size_t split, len0, len1, n;    // n = B * (len0 + len1)
  double dts[GRPO_MAX_W];         // t_{j+1} - t_j (fp64; pass 2 rounds it to fp32)
  float wb[GRPO_MAX_W], wc[GRPO_MAX_W];  // 1 - alpha_j, alpha_j
  double sigma[GRPO_MAX_W];
  const double* logp_old;         // [W][B], device
  const float* adv;               // [B], device
  float eps, adv_clip;
  // outputs: composites (mode 0) with the aggregation's split mapping, or the
  // W per-step gradients (mode 1) in the batch-B layout
  int mode;
  size_t osplit;
  void *base0, *base1, *corr0, *corr1;
  void* s_out[GRPO_MAX_W];
};
size_t grpo_part_doubles(int W, int B);
int grpo_window(const GrpoArgs& a, double* part, float* coef, double* stats, hipStream_t s);

// ---- gradient comparison: fp64 sums a.b, a.a, b.b over n elements ----
constexpr int CMP_BLOCKS = 1024;
size_t compare_part_doubles();
int grad_compare(const void* a, const void* b, size_t n, int dt, double* part, double* out_dev, hipStream_t s);
// Number of NaN / +-Inf elements of x (n elements of dt, 16-byte aligned) into
// *out_dev; part holds CMP_BLOCKS 64-bit partial counts.
int count_nonfinite(const void* x, size_t n, int dt, unsigned long long* part, unsigned long long* out_dev,
                    hipStream_t s);

}  // namespace jg
