// MMDiT forward-with-save and parameter VJP on gfx950, plus the JAGG group
// backward (Phases 3 and 4: composites, then one VJP over the batched endpoint
// pair) and the per-step baseline.  Everything is stream-ordered on the
// context's HIP stream; the caller owns every buffer.
#include <algorithm>
#include <array>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/jagg.h"
#include "attention.h"
#include "gemm.h"
#include "ops.h"
#include "prof.h"

namespace jg {

thread_local std::string g_err;
void set_error(const std::string& m) { g_err = m; }
const char* get_error() { return g_err.c_str(); }

#define TRY(x)                 \
  do {                         \
    int rc_ = (x);             \
    if (rc_) return rc_;       \
  } while (0)

struct Lin { size_t w = 0, b = 0; int out = 0, in = 0; };
struct DStream { Lin mod, qkv, o, fc1, fc2; size_t qg = 0, kg = 0; };
struct SBlock { Lin mod, in, out; size_t qg = 0, kg = 0; };

struct Model {
  dit_config c{};
  int D = 0, H = 0, Dh = 0, F = 0, C = 0, p = 0, gh = 0, gw = 0, nt = 0, ni = 0, N = 0, pd = 0, dtxt = 0, tf = 0;
  int act = F32, grad = F32;
  Lin t_in, t_out, img_in, txt_in, fmod, fin;
  std::vector<std::array<DStream, 2>> dbl;
  std::vector<SBlock> sgl;
  std::vector<jagg_tensor_desc> layout;
  size_t total = 0;
};

static size_t add_t(Model& m, const std::string& name, int rows, int cols) {
  jagg_tensor_desc d;
  std::memset(&d, 0, sizeof(d));
  std::strncpy(d.name, name.c_str(), sizeof(d.name) - 1);
  d.offset = m.total;
  d.numel = (size_t)rows * cols;
  d.rows = rows;
  d.cols = cols;
  m.layout.push_back(d);
  m.total += (d.numel + 127) / 128 * 128;
  return d.offset;
}
static Lin add_lin(Model& m, const std::string& pre, int out, int in) {
  Lin l;
  l.out = out;
  l.in = in;
  l.w = add_t(m, pre + ".w", out, in);
  l.b = add_t(m, pre + ".b", out, 1);
  return l;
}

static int build_model(const dit_config& c, Model& m) {
  auto bad = [](const char* msg) { set_error(std::string("dit_config: ") + msg); return 1; };
  if (c.n_double < 0 || c.n_single < 0 || c.hidden <= 0 || c.heads <= 0 || c.head_dim <= 0 || c.mlp_hidden <= 0)
    return bad("sizes must be positive");
  if (c.hidden != c.heads * c.head_dim) return bad("hidden must equal heads * head_dim");
  if (c.head_dim % 4 || c.head_dim > 128) return bad("head_dim must be a multiple of 4 and <= 128");
  if (c.hidden > 4096) return bad("hidden must be <= 4096");
  if (c.t_freq_dim <= 0 || c.t_freq_dim % 2) return bad("t_freq_dim must be positive and even");
  if (c.patch <= 0 || c.lat_h % c.patch || c.lat_w % c.patch) return bad("latent size must be a multiple of patch");
  if (c.in_ch <= 0 || c.lat_h <= 0 || c.lat_w <= 0 || c.n_txt <= 0) return bad("latent/text sizes must be positive");
  if (!c.block_only && c.txt_dim <= 0) return bad("txt_dim must be positive");
  if (c.block_only && c.n_single) return bad("a block-only model has double-stream blocks only");
  if (c.n_double + c.n_single == 0 && c.block_only) return bad("no blocks");
  if ((c.act_dtype != JAGG_F32 && c.act_dtype != JAGG_BF16) || (c.grad_dtype != JAGG_F32 && c.grad_dtype != JAGG_BF16))
    return bad("unknown dtype");
  m = Model();
  m.c = c;
  m.D = c.hidden; m.H = c.heads; m.Dh = c.head_dim; m.F = c.mlp_hidden;
  m.C = c.in_ch; m.p = c.patch; m.gh = c.lat_h / c.patch; m.gw = c.lat_w / c.patch;
  m.nt = c.n_txt; m.ni = m.gh * m.gw; m.N = m.nt + m.ni; m.pd = c.in_ch * c.patch * c.patch;
  m.dtxt = c.txt_dim; m.tf = c.t_freq_dim; m.act = c.act_dtype; m.grad = c.grad_dtype;
  const int D = m.D, F = m.F;
  m.t_in = add_lin(m, "t_in", D, m.tf);
  m.t_out = add_lin(m, "t_out", D, D);
  if (!c.block_only) {
    m.img_in = add_lin(m, "img_in", D, m.pd);
    m.txt_in = add_lin(m, "txt_in", D, m.dtxt);
  }
  for (int i = 0; i < c.n_double; ++i) {
    std::array<DStream, 2> st;
    const char* nm[2] = {"txt", "img"};
    for (int s = 0; s < 2; ++s) {
      const std::string p = "double." + std::to_string(i) + "." + nm[s] + ".";
      st[s].mod = add_lin(m, p + "mod", 6 * D, D);
      st[s].qkv = add_lin(m, p + "qkv", 3 * D, D);
      st[s].qg = add_t(m, p + "q_gain", m.Dh, 1);
      st[s].kg = add_t(m, p + "k_gain", m.Dh, 1);
      st[s].o = add_lin(m, p + "o", D, D);
      st[s].fc1 = add_lin(m, p + "fc1", F, D);
      st[s].fc2 = add_lin(m, p + "fc2", D, F);
    }
    m.dbl.push_back(st);
  }
  for (int i = 0; i < c.n_single; ++i) {
    SBlock b;
    const std::string p = "single." + std::to_string(i) + ".";
    b.mod = add_lin(m, p + "mod", 3 * D, D);
    b.in = add_lin(m, p + "in", 3 * D + F, D);
    b.qg = add_t(m, p + "q_gain", m.Dh, 1);
    b.kg = add_t(m, p + "k_gain", m.Dh, 1);
    b.out = add_lin(m, p + "out", D, D + F);
    m.sgl.push_back(b);
  }
  if (!c.block_only) {
    m.fmod = add_lin(m, "final.mod", 2 * D, D);
    m.fin = add_lin(m, "final", m.pd, D);
  }
  return 0;
}

// ------------------------------------------------------------------ buffers
struct Arena {
  char* base;
  size_t off = 0;
  explicit Arena(void* b) : base((char*)b) {}
  void* take(size_t bytes) {
    void* p = base ? base + off : nullptr;
    off += (bytes + 255) / 256 * 256;
    return p;
  }
  float* f32(size_t n) { return (float*)take(n * 4); }
};

struct DblAct {
  void *x_in = nullptr, *a1 = nullptr, *qkv = nullptr, *Qh = nullptr, *Kh = nullptr, *Vh = nullptr, *O = nullptr,
       *y1 = nullptr, *xm = nullptr, *a2 = nullptr, *pre = nullptr, *h = nullptr, *y2 = nullptr, *x_out = nullptr;
  float *mod[2] = {nullptr, nullptr}, *m1 = nullptr, *r1 = nullptr, *rq = nullptr, *rk = nullptr, *lse = nullptr,
        *m2 = nullptr, *r2 = nullptr;
};
struct SglAct {
  void *x_in = nullptr, *a = nullptr, *proj = nullptr, *Qh = nullptr, *Kh = nullptr, *Vh = nullptr, *cat = nullptr,
       *y = nullptr, *x_out = nullptr;
  float *mod = nullptr, *m = nullptr, *r = nullptr, *rq = nullptr, *rk = nullptr, *lse = nullptr;
};

struct Global {
  float *temb = nullptr, *h1 = nullptr, *sh1 = nullptr, *vec = nullptr, *mvec = nullptr;
  void *patches = nullptr, *txt = nullptr, *x0 = nullptr;
  float *fmod = nullptr, *fm = nullptr, *fr = nullptr;
  void* fa = nullptr;
};

struct Saved {
  Global g;
  std::vector<DblAct> d;
  std::vector<SglAct> s;
};

static void plan_dbl(const Model& m, Arena& a, int B, DblAct& A, bool full) {
  const size_t rows = (size_t)B * m.N, es = dsize(m.act);
  const size_t hn = (size_t)B * m.H * m.N;
  if (full) {
    A.mod[0] = a.f32((size_t)B * 6 * m.D);
    A.mod[1] = a.f32((size_t)B * 6 * m.D);
    A.m1 = a.f32(rows); A.r1 = a.f32(rows);
    A.a1 = a.take(rows * m.D * es);
    A.qkv = a.take(rows * 3 * m.D * es);
    A.rq = a.f32(rows * m.H); A.rk = a.f32(rows * m.H);
    A.Qh = a.take(hn * m.Dh * es); A.Kh = a.take(hn * m.Dh * es); A.Vh = a.take(hn * m.Dh * es);
    A.O = a.take(rows * m.D * es);
    A.lse = a.f32(hn);
    A.y1 = a.take(rows * m.D * es);
    A.xm = a.take(rows * m.D * es);
    A.m2 = a.f32(rows); A.r2 = a.f32(rows);
    A.a2 = a.take(rows * m.D * es);
    A.pre = a.take(rows * m.F * es);
    A.h = a.take(rows * m.F * es);
    A.y2 = a.take(rows * m.D * es);
  }
  A.x_out = a.take(rows * m.D * es);
}

static void plan_sgl(const Model& m, Arena& a, int B, SglAct& A, bool full) {
  const size_t rows = (size_t)B * m.N, es = dsize(m.act);
  const size_t hn = (size_t)B * m.H * m.N;
  if (full) {
    A.mod = a.f32((size_t)B * 3 * m.D);
    A.m = a.f32(rows); A.r = a.f32(rows);
    A.a = a.take(rows * m.D * es);
    A.proj = a.take(rows * (3 * m.D + m.F) * es);
    A.rq = a.f32(rows * m.H); A.rk = a.f32(rows * m.H);
    A.Qh = a.take(hn * m.Dh * es); A.Kh = a.take(hn * m.Dh * es); A.Vh = a.take(hn * m.Dh * es);
    A.cat = a.take(rows * (m.D + m.F) * es);
    A.lse = a.f32(hn);
    A.y = a.take(rows * m.D * es);
  }
  A.x_out = a.take(rows * m.D * es);
}

static size_t plan_saved(const Model& m, int B, void* base, Saved& S) {
  Arena a(base);
  const size_t rows = (size_t)B * m.N, es = dsize(m.act);
  S = Saved();
  S.g.temb = a.f32((size_t)B * m.tf);
  S.g.h1 = a.f32((size_t)B * m.D);
  S.g.sh1 = a.f32((size_t)B * m.D);
  S.g.vec = a.f32((size_t)B * m.D);
  S.g.mvec = a.f32((size_t)B * m.D);
  if (!m.c.block_only) {
    S.g.patches = a.take((size_t)B * m.ni * m.pd * es);
    S.g.txt = a.take((size_t)B * m.nt * m.dtxt * es);
  }
  S.g.x0 = a.take(rows * m.D * es);
  const bool full = !m.c.checkpoint;
  S.d.resize(m.c.n_double);
  S.s.resize(m.c.n_single);
  void* prev = S.g.x0;
  for (auto& A : S.d) { plan_dbl(m, a, B, A, full); A.x_in = prev; prev = A.x_out; }
  for (auto& A : S.s) { plan_sgl(m, a, B, A, full); A.x_in = prev; prev = A.x_out; }
  if (!m.c.block_only) {
    S.g.fmod = a.f32((size_t)B * 2 * m.D);
    S.g.fm = a.f32(rows);
    S.g.fr = a.f32(rows);
    S.g.fa = a.take(rows * m.D * es);
  }
  return a.off;
}

struct Ws {
  DblAct sd;
  SglAct ss;
  void *xa = nullptr, *xb = nullptr;
  float* g = nullptr;
  void* dY = nullptr;
  void* dbig = nullptr;
  float* dA = nullptr;
  void* dO = nullptr;
  void *dQh = nullptr, *dKh = nullptr, *dVh = nullptr;
  float* delta = nullptr;
  void* dS = nullptr;  // dS^T of the attention backward (bf16 MFMA path)
  float *p1 = nullptr, *p2 = nullptr;
  float* pr = nullptr;  // double block: partials of the reductions on the weight-gradient stream
  float* dmod[2] = {nullptr, nullptr};
  float *dmvec = nullptr, *dvec = nullptr, *dsh1 = nullptr, *tmp = nullptr;
  float* slpart = nullptr;
  void* gact = nullptr;
  void* fout = nullptr;
  float* dfa = nullptr;
  void* cot = nullptr;
  double *spart = nullptr, *score = nullptr;
  float* gcoef = nullptr;  // GRPO coefficients [W][B]
  int maxcols = 0;
};

static size_t out_elems(const Model& m) {  // per sample
  return m.c.block_only ? (size_t)m.N * m.D : (size_t)m.C * m.c.lat_h * m.c.lat_w;
}

// Partials of the double block's reductions that run on the weight-gradient
// stream, one region per producer (none is reused within the block):
// MLP gate (2 x [nch][D]), fc1 bias ([nch][F]), second LayerNorm (2 x [nlb][D]),
// attention gate (2 x [nch][D]), q/k gains ([nch * QK_PARTS][2 Dh]), qkv bias
// ([nch][3D]); nch chunks of RED_ROWS rows, nlb of LN_ROWS rows.
static size_t dbl_side_part_floats(const Model& m, int B) {
  const size_t nch = Chunks{B, m.nt, m.ni, RED_ROWS}.count(), nlb = Chunks{B, m.nt, m.ni, LN_ROWS}.count();
  return nch * (4 * (size_t)m.D + m.F + QK_PARTS * 2 * (size_t)m.Dh + 3 * (size_t)m.D) + 2 * nlb * m.D;
}

static size_t plan_ws(const Model& m, int B, void* base, Ws& W) {
  Arena a(base);
  const size_t rows = (size_t)B * m.N, es = dsize(m.act);
  const size_t hn = (size_t)B * m.H * m.N;
  W = Ws();
  // group-score buffers first: their offset does not depend on the batch
  W.spart = (double*)a.take(std::max({score_part_doubles(8), compare_part_doubles(),
                                       grpo_part_doubles(GRPO_MAX_W, 32)}) * sizeof(double));
  W.score = (double*)a.take(64);
  W.gcoef = (float*)a.take((size_t)GRPO_MAX_W * 32 * sizeof(float));
  if (m.c.n_double) plan_dbl(m, a, B, W.sd, true);
  if (m.c.n_single) plan_sgl(m, a, B, W.ss, true);
  W.xa = a.take(rows * m.D * es);
  W.xb = a.take(rows * m.D * es);
  W.g = a.f32(rows * m.D);
  W.dY = a.take(rows * m.D * es);
  const int big = std::max(m.F, 3 * m.D + (m.c.n_single ? m.F : 0));
  W.dbig = a.take(rows * big * es);
  W.dA = a.f32(rows * m.D);
  W.dO = a.take(rows * m.D * es);
  W.dQh = a.take(hn * m.Dh * es);
  W.dKh = a.take(hn * m.Dh * es);
  W.dVh = a.take(hn * m.Dh * es);
  W.delta = a.f32(2 * hn);  // delta, then the log-sum-exp in log2 units
  if (m.act == BF16 && m.Dh == 128)
    W.dS = a.take((size_t)B * m.H * attn_ds_rows(m.N) * attn_ds_ld(m.N) * 2);
  // per 32-row chunk: the widest partials of one launch (the LayerNorm
  // backward's come per block of LN_ROWS rows, RED_ROWS / LN_ROWS per chunk)
  W.maxcols = std::max({3 * m.D + m.F, m.D + m.F, QK_PARTS * 2 * m.Dh, RED_ROWS / LN_ROWS * m.D, m.pd});
  const int nch = Chunks{B, m.nt, m.ni, RED_ROWS}.count();
  W.p1 = a.f32((size_t)nch * W.maxcols);
  W.p2 = a.f32((size_t)nch * W.maxcols);
  if (m.c.n_double) W.pr = a.f32(dbl_side_part_floats(m, B));
  W.dmod[0] = a.f32((size_t)B * 6 * m.D);
  W.dmod[1] = a.f32((size_t)B * 6 * m.D);
  W.dmvec = a.f32((size_t)B * m.D);
  W.dvec = a.f32((size_t)B * m.D);
  W.dsh1 = a.f32((size_t)B * m.D);
  W.tmp = a.f32((size_t)B * m.D);
  // partials of every small-linear backward with an input gradient: the
  // modulations (D -> 6D or 3D or 2D) and the second time-MLP layer (D -> D)
  const size_t slp = std::max({small_linear_bwd_part_floats(B, m.D, 6 * m.D), small_linear_bwd_part_floats(B, m.D, 3 * m.D),
                               small_linear_bwd_part_floats(B, m.D, 2 * m.D), small_linear_bwd_part_floats(B, m.D, m.D),
                               small_linear_bwd_part_floats(B, m.tf, m.D)});
  W.slpart = a.f32(slp);
  W.gact = a.take(rows * m.D * es);
  if (!m.c.block_only) {
    W.fout = a.take((size_t)B * m.ni * m.pd * es);
    W.dfa = a.f32(rows * m.D);
  }
  W.cot = a.take((size_t)B * out_elems(m) * es);
  return a.off;
}

}  // namespace jg

using namespace jg;

struct jagg_ctx {
  Model m;
  hipStream_t stream = nullptr;
  void* ws = nullptr;
  size_t ws_bytes = 0;
  // second stream for the weight-gradient products of the backward, created on
  // first use (default priority), with its fork and join events
  hipStream_t side = nullptr;
  hipEvent_t fork = nullptr, join = nullptr, mark = nullptr;
};

namespace jg {

// ------------------------------------------------------------ GEMM helpers
struct Ctx {
  const Model& m;
  hipStream_t s;
  const char* th;  // theta base
  size_t es;       // theta element size
  // weight-gradient stream of the backward (nullptr: everything on s) and
  // its fork / join events
  hipStream_t side = nullptr;
  hipEvent_t ev_fork = nullptr, ev_join = nullptr, ev_mark = nullptr;
  const void* P(size_t off) const { return th + off * es; }
  // the stream the next weight-gradient product goes to: the side stream,
  // after everything issued on s so far
  hipStream_t fork() const {
    if (!side) return s;
    if (hipEventRecord(ev_fork, s) != hipSuccess || hipStreamWaitEvent(side, ev_fork, 0) != hipSuccess) return s;
    return side;
  }
  // mark(): an event after the work issued on the side stream so far;
  // wait_mark(): s waits for that work only (not for what was issued later)
  int mark() const {
    if (!side) return 0;
    if (hipEventRecord(ev_mark, side) != hipSuccess) {
      set_error("backward: marking the weight-gradient stream failed");
      return 3;
    }
    return 0;
  }
  int wait_mark() const {
    if (!side) return 0;
    if (hipStreamWaitEvent(s, ev_mark, 0) != hipSuccess) {
      set_error("backward: waiting for the weight-gradient stream failed");
      return 3;
    }
    return 0;
  }
  // s waits for every weight-gradient product issued so far
  int join() const {
    if (!side) return 0;
    if (hipEventRecord(ev_join, side) != hipSuccess || hipStreamWaitEvent(s, ev_join, 0) != hipSuccess) {
      set_error("backward: joining the weight-gradient stream failed");
      return 3;
    }
    return 0;
  }
};

// Y[M][:] = X[M][K] W[rows w_row0..][K]^T + b  (one linear layer or a row slice of it)
static GemmArgs lin_args(const Ctx& cx, const void* X, int ldx, int M, const Lin& L, int w_row0, int nout, void* Y,
                         int ldy, int mode = EPI_STORE, void* aux = nullptr, int ldaux = 0) {
  GemmArgs g;
  g.A = X; g.lda = ldx; g.ta = 0; g.a_dt = cx.m.act;
  g.B = (const char*)cx.P(L.w) + (size_t)w_row0 * L.in * cx.es; g.ldb = L.in; g.tb = 0; g.b_dt = cx.m.act;
  g.M = M; g.N = nout; g.K = L.in;
  g.epi.C = Y; g.epi.ldc = ldy; g.epi.c_dt = cx.m.act;
  g.epi.bias = (const char*)cx.P(L.b) + (size_t)w_row0 * cx.es; g.epi.bias_dt = cx.m.act;
  g.epi.mode = mode; g.epi.aux = aux; g.epi.ldaux = ldaux; g.epi.aux_dt = cx.m.act;
  return g;
}
static int lin_fwd(const Ctx& cx, const void* X, int ldx, int M, const Lin& L, int w_row0, int nout, void* Y,
                   int ldy, int mode = EPI_STORE, void* aux = nullptr, int ldaux = 0) {
  return gemm(lin_args(cx, X, ldx, M, L, w_row0, nout, Y, ldy, mode, aux, ldaux), cx.s);
}

// dW[Nout][Kin] = beta dW + dY[rows][Nout]^T X[rows][Kin]
static int wgrad(const Ctx& cx, const void* dY, int ld_dy, int dy_dt, const void* X, int ldx, int rows, int Nout,
                 int Kin, void* dW, float beta) {
  GemmArgs g;
  g.A = dY; g.lda = ld_dy; g.ta = 1; g.a_dt = dy_dt;
  g.B = X; g.ldb = ldx; g.tb = 1; g.b_dt = cx.m.act;
  g.M = Nout; g.N = Kin; g.K = rows;
  g.epi.C = dW; g.epi.ldc = Kin; g.epi.c_dt = cx.m.grad; g.epi.beta = beta;
  return gemm(g, cx.s);
}

// out[rows][Kin] = dY[rows][Nout] W[Nout][Kin] (W row-sliced via w_off/ldw) with epilogue
static int dgrad(const Ctx& cx, const void* dY, int ld_dy, int rows, const void* W, int ldw, int Nout, int Kin,
                 void* out, int ldo, int odt, int mode = EPI_STORE, void* aux = nullptr, int ldaux = 0) {
  GemmArgs g;
  g.A = dY; g.lda = ld_dy; g.ta = 0; g.a_dt = cx.m.act;
  g.B = W; g.ldb = ldw; g.tb = 1; g.b_dt = cx.m.act;
  g.M = rows; g.N = Kin; g.K = Nout;
  g.epi.C = out; g.epi.ldc = ldo; g.epi.c_dt = odt;
  g.epi.mode = mode; g.epi.aux = aux; g.epi.ldaux = ldaux; g.epi.aux_dt = cx.m.act;
  return gemm(g, cx.s);
}

static void* G(void* dth, const Model& m, size_t off) { return (char*)dth + off * dsize(m.grad); }

// -------------------------------------------------------------- forward
static int dbl_fwd(const Ctx& cx, int i, const DblAct& A, const float* mvec, int B) {
  const Model& m = cx.m;
  const int D = m.D, F = m.F;
  const RowMap rm{B, m.nt, m.ni};
  const int rt = rm.rows_txt(), R = rm.rows();
  const int r0[2] = {0, rt}, nr[2] = {rt, R - rt};
  const size_t es = dsize(m.act);
  auto row = [&](void* p, int r, int ld) { return (void*)((char*)p + (size_t)r * ld * es); };
  const auto& st = m.dbl[i];
  for (int s = 0; s < 2; ++s)
    TRY(small_linear_fwd(mvec, 0, B, D, cx.P(st[s].mod.w), cx.P(st[s].mod.b), m.act, A.mod[s], 6 * D, cx.s));
  TRY(ln_mod_fwd(A.x_in, m.act, D, rm, 0, R, A.mod[0], A.mod[1], 6 * D, 0, D, A.a1, A.m1, A.r1, cx.s));
  // the two streams' products of each layer: one grouped launch
  auto fwd2 = [&](void* X, int ldx, const Lin& L0, const Lin& L1, int nout, void* Y, int ldy, int mode = EPI_STORE,
                  void* aux = nullptr, int ldaux = 0) {
    const GemmArgs a = lin_args(cx, row(X, r0[0], ldx), ldx, nr[0], L0, 0, nout, row(Y, r0[0], ldy), ldy, mode,
                                aux ? row(aux, r0[0], ldaux) : nullptr, ldaux);
    const GemmArgs b = lin_args(cx, row(X, r0[1], ldx), ldx, nr[1], L1, 0, nout, row(Y, r0[1], ldy), ldy, mode,
                                aux ? row(aux, r0[1], ldaux) : nullptr, ldaux);
    return gemm2(a, b, cx.s);
  };
  TRY(fwd2(A.a1, D, st[0].qkv, st[1].qkv, 3 * D, A.qkv, 3 * D));
  Gains gn{{cx.P(st[0].qg), cx.P(st[1].qg)}, {cx.P(st[0].kg), cx.P(st[1].kg)}};
  TRY(qk_norm_rope_fwd(A.qkv, 3 * D, m.act, rm, Rope{m.H, m.Dh, m.nt, m.ni, m.gw}, gn, A.Qh, A.Kh, A.Vh, A.rq, A.rk,
                       cx.s));
  AttnFwd af{A.Qh, A.Kh, A.Vh, A.O, D, A.lse, B, m.H, m.N, m.Dh, m.act, rm};
  TRY(attention_fwd(af, cx.s));
  TRY(fwd2(A.O, D, st[0].o, st[1].o, D, A.y1, D));
  TRY(gated_residual(A.x_in, A.y1, m.act, D, D, rm, 0, R, A.mod[0], A.mod[1], 6 * D, 2 * D, A.xm, cx.s));
  TRY(ln_mod_fwd(A.xm, m.act, D, rm, 0, R, A.mod[0], A.mod[1], 6 * D, 3 * D, 4 * D, A.a2, A.m2, A.r2, cx.s));
  TRY(fwd2(A.a2, D, st[0].fc1, st[1].fc1, F, A.h, F, EPI_GELU_FWD, A.pre, F));
  TRY(fwd2(A.h, F, st[0].fc2, st[1].fc2, D, A.y2, D));
  TRY(gated_residual(A.xm, A.y2, m.act, D, D, rm, 0, R, A.mod[0], A.mod[1], 6 * D, 5 * D, A.x_out, cx.s));
  return 0;
}

static int sgl_fwd(const Ctx& cx, int i, const SglAct& A, const float* mvec, int B) {
  const Model& m = cx.m;
  const int D = m.D, F = m.F, LD = 3 * D + F, LC = D + F;
  const RowMap rm{B, m.nt, m.ni};
  const int R = rm.rows();
  const size_t es = dsize(m.act);
  const SBlock& sb = m.sgl[i];
  TRY(small_linear_fwd(mvec, 0, B, D, cx.P(sb.mod.w), cx.P(sb.mod.b), m.act, A.mod, 3 * D, cx.s));
  TRY(ln_mod_fwd(A.x_in, m.act, D, rm, 0, R, A.mod, A.mod, 3 * D, 0, D, A.a, A.m, A.r, cx.s));
  TRY(lin_fwd(cx, A.a, D, R, sb.in, 0, 3 * D, A.proj, LD));
  TRY(lin_fwd(cx, A.a, D, R, sb.in, 3 * D, F, (char*)A.cat + D * es, LC, EPI_GELU_FWD, (char*)A.proj + 3 * D * es,
              LD));
  Gains gn{{cx.P(sb.qg), cx.P(sb.qg)}, {cx.P(sb.kg), cx.P(sb.kg)}};
  TRY(qk_norm_rope_fwd(A.proj, LD, m.act, rm, Rope{m.H, m.Dh, m.nt, m.ni, m.gw}, gn, A.Qh, A.Kh, A.Vh, A.rq, A.rk,
                       cx.s));
  AttnFwd af{A.Qh, A.Kh, A.Vh, A.cat, LC, A.lse, B, m.H, m.N, m.Dh, m.act, rm};
  TRY(attention_fwd(af, cx.s));
  TRY(lin_fwd(cx, A.cat, LC, R, sb.out, 0, D, A.y, D));
  TRY(gated_residual(A.x_in, A.y, m.act, D, D, rm, 0, R, A.mod, A.mod, 3 * D, 2 * D, A.x_out, cx.s));
  return 0;
}

static int forward(jagg_ctx* ctx, const void* theta, const void* z, const float* t, const void* txt, void* v_out,
                   void* saved, int B) {
  const Model& m = ctx->m;
  Ctx cx{m, ctx->stream, (const char*)theta, dsize(m.act)};
  const size_t es = dsize(m.act);
  const RowMap rm{B, m.nt, m.ni};
  const int rt = rm.rows_txt(), R = rm.rows(), D = m.D;
  Ws W;
  plan_ws(m, B, ctx->ws, W);
  Saved S;
  Saved* SP = nullptr;
  if (saved) { plan_saved(m, B, saved, S); SP = &S; }
  // global activations live in `saved`, or in the workspace scratch otherwise
  Global gl;
  if (SP) gl = S.g;
  else {
    Saved tmp;
    // no-grad: borrow workspace regions (gradient buffers are idle in a forward)
    gl.temb = W.dA; gl.h1 = W.dvec; gl.sh1 = W.dsh1; gl.vec = W.tmp; gl.mvec = W.dmvec;
    gl.patches = W.dbig;
    gl.txt = (char*)W.dbig + (size_t)B * m.ni * m.pd * es;
    gl.x0 = W.xa;
    gl.fmod = W.dmod[0]; gl.fm = W.p1; gl.fr = W.p2; gl.fa = W.gact;
    (void)tmp;
  }
  TVals tv;
  for (int b = 0; b < B; ++b) tv.t[b] = t[b];
  TRY(time_embed(tv, B, m.tf, gl.temb, cx.s));
  TRY(small_linear_fwd(gl.temb, 0, B, m.tf, cx.P(m.t_in.w), cx.P(m.t_in.b), m.act, gl.h1, D, cx.s));
  TRY(silu_fwd(gl.h1, gl.sh1, (size_t)B * D, cx.s));
  TRY(small_linear_fwd(gl.sh1, 0, B, D, cx.P(m.t_out.w), cx.P(m.t_out.b), m.act, gl.vec, D, cx.s));
  TRY(silu_fwd(gl.vec, gl.mvec, (size_t)B * D, cx.s));
  if (m.c.block_only) {
    if (hipMemcpyAsync(gl.x0, z, (size_t)R * D * es, hipMemcpyDeviceToDevice, cx.s) != hipSuccess) {
      set_error("forward: copy of the input token rows failed");
      return 3;
    }
  } else {
    TRY(patchify(z, m.act, B, m.C, m.c.lat_h, m.c.lat_w, m.p, gl.patches, cx.s));
    TRY(lin_fwd(cx, gl.patches, m.pd, B * m.ni, m.img_in, 0, D, (char*)gl.x0 + (size_t)rt * D * es, D));
    if (hipMemcpyAsync(gl.txt, txt, (size_t)B * m.nt * m.dtxt * es, hipMemcpyDeviceToDevice, cx.s) != hipSuccess) {
      set_error("forward: copy of the text embeddings failed");
      return 3;
    }
    TRY(lin_fwd(cx, gl.txt, m.dtxt, rt, m.txt_in, 0, D, gl.x0, D));
  }
  const bool keep = SP && !m.c.checkpoint;
  void* x = gl.x0;
  int pp = 0;
  for (int i = 0; i < m.c.n_double; ++i) {
    DblAct A = keep ? S.d[i] : W.sd;
    A.x_in = x;
    if (SP) A.x_out = S.d[i].x_out;
    else A.x_out = (pp++ % 2) ? W.xa : W.xb;
    TRY(dbl_fwd(cx, i, A, gl.mvec, B));
    x = A.x_out;
  }
  for (int i = 0; i < m.c.n_single; ++i) {
    SglAct A = keep ? S.s[i] : W.ss;
    A.x_in = x;
    if (SP) A.x_out = S.s[i].x_out;
    else A.x_out = (pp++ % 2) ? W.xa : W.xb;
    TRY(sgl_fwd(cx, i, A, gl.mvec, B));
    x = A.x_out;
  }
  if (m.c.block_only) {
    if (hipMemcpyAsync(v_out, x, (size_t)R * D * es, hipMemcpyDeviceToDevice, cx.s) != hipSuccess) {
      set_error("forward: copy of the output token rows failed");
      return 3;
    }
    return 0;
  }
  TRY(small_linear_fwd(gl.mvec, 0, B, D, cx.P(m.fmod.w), cx.P(m.fmod.b), m.act, gl.fmod, 2 * D, cx.s));
  TRY(ln_mod_fwd(x, m.act, D, rm, rt, R - rt, gl.fmod, gl.fmod, 2 * D, 0, D, gl.fa, gl.fm, gl.fr, cx.s));
  TRY(lin_fwd(cx, (char*)gl.fa + (size_t)rt * D * es, D, B * m.ni, m.fin, 0, m.pd, W.fout, m.pd));
  TRY(unpatchify(W.fout, m.act, B, m.C, m.c.lat_h, m.c.lat_w, m.p, v_out, cx.s));
  return 0;
}

// ------------------------------------------------------------------ VJP
// The text- and image-stream products of one layer of a double block (separate
// weights, disjoint row ranges) as one grouped GEMM launch.
static GemmArgs wgrad_args(const Ctx& cx, const void* dY, int ld_dy, int dy_dt, const void* X, int ldx, int rows,
                           int Nout, int Kin, void* dW, float beta) {
  GemmArgs g;
  g.A = dY; g.lda = ld_dy; g.ta = 1; g.a_dt = dy_dt;
  g.B = X; g.ldb = ldx; g.tb = 1; g.b_dt = cx.m.act;
  g.M = Nout; g.N = Kin; g.K = rows;
  g.epi.C = dW; g.epi.ldc = Kin; g.epi.c_dt = cx.m.grad; g.epi.beta = beta;
  return g;
}
static GemmArgs dgrad_args(const Ctx& cx, const void* dY, int ld_dy, int rows, const void* W, int ldw, int Nout,
                           int Kin, void* out, int ldo, int odt, int mode = EPI_STORE, void* aux = nullptr,
                           int ldaux = 0) {
  GemmArgs g;
  g.A = dY; g.lda = ld_dy; g.ta = 0; g.a_dt = cx.m.act;
  g.B = W; g.ldb = ldw; g.tb = 1; g.b_dt = cx.m.act;
  g.M = rows; g.N = Kin; g.K = Nout;
  g.epi.C = out; g.epi.ldc = ldo; g.epi.c_dt = odt;
  g.epi.mode = mode; g.epi.aux = aux; g.epi.ldaux = ldaux; g.epi.aux_dt = cx.m.act;
  return g;
}

// Double-block backward.  Both streams' rows go through every memory-bound
// kernel in one launch (the modulation vectors are picked per row), and the
// two streams' products of each layer run as one grouped GEMM; only the
// per-stream reductions of the column partials are separate launches.
// gin (gin_dt): the gradient arriving at the block's output, W.g itself or
// (the model's first backward block) the cotangent in the activation dtype;
// W.g holds the gradient at the block's input on return.
static int dbl_bwd(const Ctx& cx, int i, const DblAct& A, const float* mvec, int B, Ws& W, void* dth, float beta,
                   const void* gin, int gin_dt) {
  const Model& m = cx.m;
  const int D = m.D, F = m.F, act = m.act;
  const RowMap rm{B, m.nt, m.ni};
  const int rt = rm.rows_txt(), R = rm.rows();
  const int r0[2] = {0, rt}, nr[2] = {rt, R - rt};
  const size_t es = dsize(act);
  auto row = [&](void* p, int r, int ld) { return (void*)((char*)p + (size_t)r * ld * es); };
  auto rowf = [&](float* p, int r, int ld) { return p + (size_t)r * ld; };
  const auto& st = m.dbl[i];
  const int nchunk = Chunks{B, m.nt, m.ni, RED_ROWS}.count();
  int c0[2], nc[2];
  for (int s = 0; s < 2; ++s) TRY(chunk_range(rm, r0[s], nr[s], &c0[s], &nc[s]));
  const hipStream_t S = cx.s;
  // regions of the reductions that go to the weight-gradient stream (their
  // results are needed only at the block's end): MLP gate, fc1 bias, second
  // LayerNorm, attention gate, q/k gains, qkv bias
  const size_t nch = nchunk, nlb = Chunks{B, m.nt, m.ni, LN_ROWS}.count();
  float* const g2a = W.pr;
  float* const g2b = g2a + nch * D;
  float* const cf1 = g2b + nch * D;
  float* const l2a = cf1 + nch * F;
  float* const l2b = l2a + nlb * D;
  float* const g1a = l2b + nlb * D;
  float* const g1b = g1a + nch * D;
  float* const qkg = g1b + nch * D;
  float* const cqkv = qkg + nch * QK_PARTS * 2 * m.Dh;
  auto wg2 = [&](void* dY, int ld_dy, void* X, int ldx, int Nout, int Kin, size_t w0, size_t w1) {
    const GemmArgs a = wgrad_args(cx, row(dY, r0[0], ld_dy), ld_dy, act, row(X, r0[0], ldx), ldx, nr[0], Nout, Kin,
                                  G(dth, m, w0), beta);
    const GemmArgs b = wgrad_args(cx, row(dY, r0[1], ld_dy), ld_dy, act, row(X, r0[1], ldx), ldx, nr[1], Nout, Kin,
                                  G(dth, m, w1), beta);
    // weight gradients feed nothing later in the pass: they go to the
    // weight-gradient stream, which s joins before dY's buffer is reused
    return gemm2(a, b, cx.fork());
  };
  auto dg2 = [&](void* dY, int ld_dy, size_t w0, size_t w1, int ldw, int Nout, int Kin, void* out, int ldo, int odt,
                 int mode = EPI_STORE, void* aux = nullptr, int ldaux = 0) {
    const size_t oes = dsize(odt);
    auto orow = [&](void* p, int r) { return (void*)((char*)p + (size_t)r * ldo * oes); };
    const GemmArgs a = dgrad_args(cx, row(dY, r0[0], ld_dy), ld_dy, nr[0], cx.P(w0), ldw, Nout, Kin, orow(out, r0[0]),
                                  ldo, odt, mode, aux ? row(aux, r0[0], ldaux) : nullptr, ldaux);
    const GemmArgs b = dgrad_args(cx, row(dY, r0[1], ld_dy), ld_dy, nr[1], cx.P(w1), ldw, Nout, Kin, orow(out, r0[1]),
                                  ldo, odt, mode, aux ? row(aux, r0[1], ldaux) : nullptr, ldaux);
    return gemm2(a, b, S);
  };
  // MLP branch: x_out = xm + gate2 * y2
  TRY(gate_bwd(gin, gin_dt, A.y2, act, D, rm, 0, R, A.mod[0], A.mod[1], 6 * D, 5 * D, W.dY, D, g2a, g2b, S));
  {
    RedJob j[4];
    for (int s = 0; s < 2; ++s) {
      j[s] = per_sample_job(g2a, D, rm, r0[s], nr[s], W.dmod[s], 6 * D, 5 * D);
      j[2 + s] = to_grad_job(g2b, D, c0[s], nc[s], D, G(dth, m, st[s].fc2.b), m.grad, beta);
    }
    TRY(reduce_jobs(j, 4, cx.fork()));
  }
  TRY(wg2(W.dY, D, A.h, F, D, F, st[0].fc2.w, st[1].fc2.w));
  TRY(dg2(W.dY, D, st[0].fc2.w, st[1].fc2.w, F, D, F, W.dbig, F, act, EPI_GELU_BWD, A.pre, F));
  TRY(colsum_partials(W.dbig, act, F, F, rm, 0, R, cf1, S));
  {
    RedJob j[2];
    for (int s = 0; s < 2; ++s) j[s] = to_grad_job(cf1, F, c0[s], nc[s], F, G(dth, m, st[s].fc1.b), m.grad, beta);
    TRY(reduce_jobs(j, 2, cx.fork()));
  }
  TRY(wg2(W.dbig, F, A.a2, D, F, D, st[0].fc1.w, st[1].fc1.w));
  TRY(dg2(W.dbig, F, st[0].fc1.w, st[1].fc1.w, D, F, D, W.dA, D, F32));
  TRY(ln_mod_bwd(W.dA, A.xm, act, D, rm, 0, R, A.m2, A.r2, A.mod[0], A.mod[1], 6 * D, 4 * D, gin, gin_dt, W.g, l2a,
                 l2b, S));
  {
    RedJob j[4];
    for (int s = 0; s < 2; ++s) {
      j[2 * s] = per_sample_job(l2a, D, rm, r0[s], nr[s], W.dmod[s], 6 * D, 4 * D, LN_ROWS);
      j[2 * s + 1] = per_sample_job(l2b, D, rm, r0[s], nr[s], W.dmod[s], 6 * D, 3 * D, LN_ROWS);
    }
    TRY(reduce_jobs(j, 4, cx.fork()));
  }
  // attention branch: xm = x + gate1 * y1 (W.dY and W.dbig are rewritten
  // from here on: the fc2 and fc1 weight gradients that read them are done)
  TRY(cx.join());
  TRY(gate_bwd(W.g, F32, A.y1, act, D, rm, 0, R, A.mod[0], A.mod[1], 6 * D, 2 * D, W.dY, D, g1a, g1b, S));
  {
    RedJob j[4];
    for (int s = 0; s < 2; ++s) {
      j[s] = per_sample_job(g1a, D, rm, r0[s], nr[s], W.dmod[s], 6 * D, 2 * D);
      j[2 + s] = to_grad_job(g1b, D, c0[s], nc[s], D, G(dth, m, st[s].o.b), m.grad, beta);
    }
    TRY(reduce_jobs(j, 4, cx.fork()));
    // the last modulation sums on that stream: the block's end waits for them
    TRY(cx.mark());
  }
  TRY(wg2(W.dY, D, A.O, D, D, D, st[0].o.w, st[1].o.w));
  TRY(dg2(W.dY, D, st[0].o.w, st[1].o.w, D, D, D, W.dO, D, act));
  AttnBwd ab{A.Qh, A.Kh, A.Vh, A.O, D, W.dO, D, A.lse, W.delta, W.dQh, W.dKh, W.dVh, act, B, m.H, m.N, m.Dh, act, rm,
             W.dS, attn_ds_ld(m.N), attn_ds_rows(m.N)};
  TRY(attention_bwd(ab, S));
  Gains gn{{cx.P(st[0].qg), cx.P(st[1].qg)}, {cx.P(st[0].kg), cx.P(st[1].kg)}};
  TRY(qk_norm_rope_bwd(W.dQh, W.dKh, W.dVh, act, A.qkv, 3 * D, act, rm, Rope{m.H, m.Dh, m.nt, m.ni, m.gw}, gn, A.rq,
                       A.rk, W.dbig, 3 * D, qkg, S));
  // the gain partials wait for the qkv bias partials: one launch
  TRY(colsum_partials(W.dbig, act, 3 * D, 3 * D, rm, 0, R, cqkv, S));
  {
    RedJob j[6];
    for (int s = 0; s < 2; ++s) {
      j[3 * s] = to_grad_job(qkg, 2 * m.Dh, c0[s] * QK_PARTS, nc[s] * QK_PARTS, m.Dh, G(dth, m, st[s].qg), m.grad,
                             beta);
      j[3 * s + 1] = to_grad_job(qkg + m.Dh, 2 * m.Dh, c0[s] * QK_PARTS, nc[s] * QK_PARTS, m.Dh,
                                 G(dth, m, st[s].kg), m.grad, beta);
      j[3 * s + 2] = to_grad_job(cqkv, 3 * D, c0[s], nc[s], 3 * D, G(dth, m, st[s].qkv.b), m.grad, beta);
    }
    TRY(reduce_jobs(j, 6, cx.fork()));
  }
  TRY(wg2(W.dbig, 3 * D, A.a1, D, 3 * D, D, st[0].qkv.w, st[1].qkv.w));
  TRY(dg2(W.dbig, 3 * D, st[0].qkv.w, st[1].qkv.w, D, 3 * D, D, W.dA, D, F32));
  TRY(ln_mod_bwd(W.dA, A.x_in, act, D, rm, 0, R, A.m1, A.r1, A.mod[0], A.mod[1], 6 * D, D, W.g, F32, W.g, W.p1, W.p2,
                 S));
  {
    RedJob j[4];
    for (int s = 0; s < 2; ++s) {
      j[2 * s] = per_sample_job(W.p1, D, rm, r0[s], nr[s], W.dmod[s], 6 * D, D, LN_ROWS);
      j[2 * s + 1] = per_sample_job(W.p2, D, rm, r0[s], nr[s], W.dmod[s], 6 * D, 0, LN_ROWS);
    }
    TRY(reduce_jobs(j, 4, S));
  }
  // the modulation sums of the two gates and the second LayerNorm
  TRY(cx.wait_mark());
  // adaLN modulation: mod = SiLU(vec) W_mod^T + b, per stream; d SiLU(vec) in the order text, image
  for (int s = 0; s < 2; ++s) {
    TRY(small_linear_bwd(W.dmod[s], mvec, 0, B, D, cx.P(st[s].mod.w), m.act, 6 * D, G(dth, m, st[s].mod.w),
                         G(dth, m, st[s].mod.b), m.grad, beta, W.dmvec, W.slpart, S, true));
  }
  TRY(cx.join());  // the next block reuses W.dY and W.dbig
  (void)rowf;
  return 0;
}

static int sgl_bwd(const Ctx& cx, int i, const SglAct& A, const float* mvec, int B, Ws& W, void* dth, float beta) {
  const Model& m = cx.m;
  const int D = m.D, F = m.F, act = m.act, LD = 3 * D + F, LC = D + F;
  const RowMap rm{B, m.nt, m.ni};
  const int R = rm.rows();
  const size_t es = dsize(act);
  const SBlock& L = m.sgl[i];
  const int nchunk = Chunks{B, m.nt, m.ni, RED_ROWS}.count();
  TRY(gate_bwd(W.g, F32, A.y, act, D, rm, 0, R, A.mod, A.mod, 3 * D, 2 * D, W.dY, D, W.p1, W.p2, cx.s));
  {
    const RedJob j[2] = {per_sample_job(W.p1, D, rm, 0, R, W.dmod[0], 3 * D, 2 * D),
                         to_grad_job(W.p2, D, 0, nchunk, D, G(dth, m, L.out.b), m.grad, beta)};
    TRY(reduce_jobs(j, 2, cx.s));
  }
  TRY(wgrad(cx, W.dY, D, act, A.cat, LC, R, D, LC, G(dth, m, L.out.w), beta));
  // d[O, gelu(u)] = dY W_out: attention part, then the MLP part through GELU'
  TRY(dgrad(cx, W.dY, D, R, cx.P(L.out.w), LC, D, D, W.dO, D, act));
  TRY(dgrad(cx, W.dY, D, R, (const char*)cx.P(L.out.w) + (size_t)D * es, LC, D, F, (char*)W.dbig + 3 * D * es, LD,
            act, EPI_GELU_BWD, (char*)A.proj + 3 * D * es, LD));
  AttnBwd ab{A.Qh, A.Kh, A.Vh, A.cat, LC, W.dO, D, A.lse, W.delta, W.dQh, W.dKh, W.dVh, act, B, m.H, m.N, m.Dh, act, rm,
             W.dS, attn_ds_ld(m.N), attn_ds_rows(m.N)};
  TRY(attention_bwd(ab, cx.s));
  Gains gn{{cx.P(L.qg), cx.P(L.qg)}, {cx.P(L.kg), cx.P(L.kg)}};
  TRY(qk_norm_rope_bwd(W.dQh, W.dKh, W.dVh, act, A.proj, LD, act, rm, Rope{m.H, m.Dh, m.nt, m.ni, m.gw}, gn, A.rq,
                       A.rk, W.dbig, LD, W.p2, cx.s));
  // the gain partials (W.p2) wait for the input-projection bias partials (W.p1): one launch
  TRY(colsum_partials(W.dbig, act, LD, LD, rm, 0, R, W.p1, cx.s));
  {
    const RedJob j[3] = {to_grad_job(W.p2, 2 * m.Dh, 0, nchunk * QK_PARTS, m.Dh, G(dth, m, L.qg), m.grad, beta),
                         to_grad_job(W.p2 + m.Dh, 2 * m.Dh, 0, nchunk * QK_PARTS, m.Dh, G(dth, m, L.kg), m.grad, beta),
                         to_grad_job(W.p1, LD, 0, nchunk, LD, G(dth, m, L.in.b), m.grad, beta)};
    TRY(reduce_jobs(j, 3, cx.s));
  }
  TRY(wgrad(cx, W.dbig, LD, act, A.a, D, R, LD, D, G(dth, m, L.in.w), beta));
  TRY(dgrad(cx, W.dbig, LD, R, cx.P(L.in.w), D, LD, D, W.dA, D, F32));
  TRY(ln_mod_bwd(W.dA, A.x_in, act, D, rm, 0, R, A.m, A.r, A.mod, A.mod, 3 * D, D, W.g, F32, W.g, W.p1, W.p2, cx.s));
  {
    const RedJob j[2] = {per_sample_job(W.p1, D, rm, 0, R, W.dmod[0], 3 * D, D, LN_ROWS),
                         per_sample_job(W.p2, D, rm, 0, R, W.dmod[0], 3 * D, 0, LN_ROWS)};
    TRY(reduce_jobs(j, 2, cx.s));
  }
  TRY(small_linear_bwd(W.dmod[0], mvec, 0, B, D, cx.P(L.mod.w), m.act, 3 * D, G(dth, m, L.mod.w), G(dth, m, L.mod.b),
                       m.grad, beta, W.dmvec, W.slpart, cx.s, true));
  return 0;
}

// The context's weight-gradient stream and events, created on first use;
// false (everything stays on the context's stream) if any creation fails.
static bool side_stream(jagg_ctx* ctx) {
  if (ctx->side) return true;
  hipStream_t st = nullptr;
  hipEvent_t f = nullptr, j = nullptr, k = nullptr;
  if (hipStreamCreateWithFlags(&st, hipStreamNonBlocking) == hipSuccess &&
      hipEventCreateWithFlags(&f, hipEventDisableTiming) == hipSuccess &&
      hipEventCreateWithFlags(&j, hipEventDisableTiming) == hipSuccess &&
      hipEventCreateWithFlags(&k, hipEventDisableTiming) == hipSuccess) {
    ctx->side = st;
    ctx->fork = f;
    ctx->join = j;
    ctx->mark = k;
    return true;
  }
  if (k) (void)hipEventDestroy(k);
  if (j) (void)hipEventDestroy(j);
  if (f) (void)hipEventDestroy(f);
  if (st) (void)hipStreamDestroy(st);
  (void)hipGetLastError();
  return false;
}

static int vjp(jagg_ctx* ctx, const void* theta, const void* saved, int B, const void* cot, void* dth, float beta) {
  const Model& m = ctx->m;
  Ctx cx{m, ctx->stream, (const char*)theta, dsize(m.act)};
  // the double-block weight gradients overlap the rest of the pass on a second
  // stream, except while a kernel class is timed (each timed kernel runs alone)
  if (!prof_armed() && side_stream(ctx)) {
    cx.side = ctx->side;
    cx.ev_fork = ctx->fork;
    cx.ev_join = ctx->join;
    cx.ev_mark = ctx->mark;
  }
  const int act = m.act, D = m.D;
  const size_t es = dsize(act);
  const RowMap rm{B, m.nt, m.ni};
  const int rt = rm.rows_txt(), R = rm.rows();
  const int nchunk = Chunks{B, m.nt, m.ni, RED_ROWS}.count();
  Ws W;
  plan_ws(m, B, ctx->ws, W);
  Saved S;
  plan_saved(m, B, (void*)saved, S);
  const Global& gl = S.g;
  TRY(fill_zero(W.dmvec, (size_t)B * D * 4, cx.s));
  // the gradient arriving at the last block: the cotangent itself when that
  // block is a double block of a block-only model (its gate and second
  // LayerNorm backward read it in the activation dtype), else W.g
  const void* gin = W.g;
  int gin_dt = F32;
  if (m.c.block_only && m.c.n_single == 0 && m.c.n_double > 0) {
    gin = cot;
    gin_dt = act;
  } else if (m.c.block_only) {
    TRY(convert(cot, act, W.g, F32, (size_t)R * D, cx.s));
  } else {
    // final layer: v = unpatchify((LN(x_img)(1 + scale) + shift) W_f^T + b_f)
    TRY(patchify(cot, act, B, m.C, m.c.lat_h, m.c.lat_w, m.p, W.fout, cx.s));
    const int Mi = B * m.ni;
    const RowMap rimg{B, 0, m.ni};  // image rows only, as their own row space
    TRY(colsum_partials(W.fout, act, m.pd, m.pd, rimg, 0, Mi, W.p1, cx.s));
    TRY(reduce_to_grad(W.p1, m.pd, 0, Chunks{B, 0, m.ni, RED_ROWS}.count(), m.pd, G(dth, m, m.fin.b), m.grad, beta,
                       cx.s));
    TRY(wgrad(cx, W.fout, m.pd, act, (char*)gl.fa + (size_t)rt * D * es, D, Mi, m.pd, D, G(dth, m, m.fin.w), beta));
    TRY(dgrad(cx, W.fout, m.pd, Mi, cx.P(m.fin.w), D, m.pd, D, W.dfa + (size_t)rt * D, D, F32));
    TRY(fill_zero(W.g, (size_t)R * D * 4, cx.s));
    void* xl = m.sgl.empty() ? (m.dbl.empty() ? gl.x0 : S.d.back().x_out) : S.s.back().x_out;
    TRY(ln_mod_bwd(W.dfa, xl, act, D, rm, rt, R - rt, gl.fm, gl.fr, gl.fmod, gl.fmod, 2 * D, D, W.g, F32, W.g, W.p1,
                   W.p2, cx.s));
    TRY(reduce_per_sample(W.p1, D, rm, rt, R - rt, W.dmod[0], 2 * D, D, cx.s, LN_ROWS));
    TRY(reduce_per_sample(W.p2, D, rm, rt, R - rt, W.dmod[0], 2 * D, 0, cx.s, LN_ROWS));
    TRY(small_linear_bwd(W.dmod[0], gl.mvec, 0, B, D, cx.P(m.fmod.w), act, 2 * D, G(dth, m, m.fmod.w),
                         G(dth, m, m.fmod.b), m.grad, beta, W.dmvec, W.slpart, cx.s, true));
  }
  for (int i = m.c.n_single - 1; i >= 0; --i) {
    SglAct A = S.s[i];
    if (m.c.checkpoint) {
      SglAct R2 = W.ss;
      R2.x_in = S.s[i].x_in;
      R2.x_out = W.xa;
      TRY(sgl_fwd(cx, i, R2, gl.mvec, B));
      A = R2;
    }
    TRY(sgl_bwd(cx, i, A, gl.mvec, B, W, dth, beta));
  }
  for (int i = m.c.n_double - 1; i >= 0; --i) {
    DblAct A = S.d[i];
    if (m.c.checkpoint) {
      DblAct R2 = W.sd;
      R2.x_in = S.d[i].x_in;
      R2.x_out = W.xa;
      TRY(dbl_fwd(cx, i, R2, gl.mvec, B));
      A = R2;
    }
    TRY(dbl_bwd(cx, i, A, gl.mvec, B, W, dth, beta, gin, gin_dt));
    gin = W.g;
    gin_dt = F32;
  }
  if (!m.c.block_only) {
    // input embeddings (no gradient to the inputs themselves)
    TRY(convert(W.g, F32, W.gact, act, (size_t)R * D, cx.s));
    int c0, nc;
    TRY(colsum_partials(W.g, F32, D, D, rm, rt, R - rt, W.p1, cx.s));
    TRY(chunk_range(rm, rt, R - rt, &c0, &nc));
    TRY(reduce_to_grad(W.p1, D, c0, nc, D, G(dth, m, m.img_in.b), m.grad, beta, cx.s));
    TRY(wgrad(cx, (char*)W.gact + (size_t)rt * D * es, D, act, gl.patches, m.pd, B * m.ni, D, m.pd,
              G(dth, m, m.img_in.w), beta));
    TRY(colsum_partials(W.g, F32, D, D, rm, 0, rt, W.p1, cx.s));
    TRY(chunk_range(rm, 0, rt, &c0, &nc));
    TRY(reduce_to_grad(W.p1, D, c0, nc, D, G(dth, m, m.txt_in.b), m.grad, beta, cx.s));
    TRY(wgrad(cx, W.gact, D, act, gl.txt, m.dtxt, rt, D, m.dtxt, G(dth, m, m.txt_in.w), beta));
  }
  (void)nchunk;
  // time MLP: vec = SiLU(temb W1^T + b1) W2^T + b2; modulations read SiLU(vec)
  TRY(mul_silu_grad(W.dmvec, gl.vec, (size_t)B * D, cx.s));
  TRY(small_linear_bwd(W.dmvec, gl.sh1, 0, B, D, cx.P(m.t_out.w), act, D, G(dth, m, m.t_out.w), G(dth, m, m.t_out.b),
                       m.grad, beta, W.dsh1, W.slpart, cx.s));
  TRY(mul_silu_grad(W.dsh1, gl.h1, (size_t)B * D, cx.s));
  TRY(small_linear_bwd(W.dsh1, gl.temb, 0, B, m.tf, cx.P(m.t_in.w), act, D, G(dth, m, m.t_in.w), G(dth, m, m.t_in.b),
                       m.grad, beta, nullptr, W.slpart, cx.s));
  return 0;
}

}  // namespace jg

// ====================================================================== C ABI
namespace {

constexpr int MAX_BATCH = 32;

jagg_status fail(jagg_status st, const std::string& msg) {
  jg::set_error(msg);
  return st;
}

jagg_status to_status(int rc) {
  if (rc == 0) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) {
      jg::set_error(std::string("HIP error: ") + hipGetErrorString(e));
      return JAGG_EDEVICE;
    }
    return JAGG_OK;
  }
  return (jagg_status)rc;
}

// A window's (or trajectory's) timesteps run from high to low noise: strictly
// decreasing (NaN fails the comparison too).
bool decreasing(const float* t, int n) {
  for (int j = 0; j + 1 < n; ++j)
    if (!(t[j + 1] < t[j])) return false;
  return true;
}

// Gradient quality from the fp64 sums (a.b, a.a, b.b) in out[0..2]: out[3] =
// cos(a, b) = a.b / sqrt(a.a b.b), out[4] = rho = |a| / |b| (gradient-quality
// appendix); NaN where a norm is zero.
void quality_from_sums(double* out) {
  const double ab = out[0], aa = out[1], bb = out[2];
  out[3] = (aa > 0.0 && bb > 0.0) ? ab / std::sqrt(aa * bb) : std::nan("");
  out[4] = bb > 0.0 ? std::sqrt(aa / bb) : std::nan("");
}

// The batch-independent head of the workspace (reduction partials, the score
// slot, the GRPO coefficients) is all the scoring, comparison and GRPO calls
// use; it must lie inside the bound workspace.
jagg_status need_head_ws(const jagg_ctx* ctx, jg::Ws& W0, const char* who) {
  if (!ctx->ws) return fail(JAGG_EINVAL, std::string(who) + ": workspace not bound");
  jg::plan_ws(ctx->m, 1, ctx->ws, W0);
  const char* end = (const char*)W0.gcoef + (size_t)jg::GRPO_MAX_W * 32 * sizeof(float);
  if (end > (const char*)ctx->ws + ctx->ws_bytes)
    return fail(JAGG_EINVAL, std::string(who) + ": workspace smaller than its " +
                                 std::to_string(end - (const char*)ctx->ws) + "-byte head");
  return JAGG_OK;
}

jagg_status need_ws(const jagg_ctx* ctx, int batch) {
  jg::Ws W;
  const size_t need = jg::plan_ws(ctx->m, batch, nullptr, W);
  if (!ctx->ws || ctx->ws_bytes < need)
    return fail(JAGG_EINVAL, "workspace not bound or smaller than dit_workspace_bytes(" + std::to_string(batch) +
                                 ") = " + std::to_string(need));
  return JAGG_OK;
}

}  // namespace

extern "C" {

const char* jagg_last_error(void) { return jg::get_error(); }

jagg_status dit_param_layout(const dit_config* cfg, size_t* n_tensors, size_t* n_elems, jagg_tensor_desc* out,
                             size_t cap) {
  if (!cfg || !n_tensors || !n_elems) return fail(JAGG_EINVAL, "dit_param_layout: null argument");
  jg::Model m;
  if (jg::build_model(*cfg, m)) return JAGG_EINVAL;
  *n_tensors = m.layout.size();
  *n_elems = m.total;
  if (out)
    for (size_t i = 0; i < m.layout.size() && i < cap; ++i) out[i] = m.layout[i];
  return JAGG_OK;
}

jagg_status jagg_ctx_create(const dit_config* cfg, void* hip_stream, jagg_ctx** out) {
  if (!cfg || !out) return fail(JAGG_EINVAL, "jagg_ctx_create: null argument");
  jagg_ctx* c = new (std::nothrow) jagg_ctx();
  if (!c) return fail(JAGG_ENOMEM, "jagg_ctx_create: out of host memory");
  if (jg::build_model(*cfg, c->m)) { delete c; return JAGG_EINVAL; }
  c->stream = (hipStream_t)hip_stream;
  *out = c;
  return JAGG_OK;
}

void jagg_ctx_destroy(jagg_ctx* ctx) {
  if (!ctx) return;
  if (ctx->side) {
    (void)hipStreamSynchronize(ctx->side);
    (void)hipEventDestroy(ctx->fork);
    (void)hipEventDestroy(ctx->join);
    (void)hipEventDestroy(ctx->mark);
    (void)hipStreamDestroy(ctx->side);
  }
  delete ctx;
}

jagg_status dit_saved_bytes(const jagg_ctx* ctx, int batch, size_t* bytes) {
  if (!ctx || !bytes) return fail(JAGG_EINVAL, "dit_saved_bytes: null argument");
  if (batch < 1 || batch > MAX_BATCH) return fail(JAGG_EINVAL, "dit_saved_bytes: batch must be 1..32");
  jg::Saved S;
  *bytes = jg::plan_saved(ctx->m, batch, nullptr, S);
  return JAGG_OK;
}

jagg_status dit_workspace_bytes(const jagg_ctx* ctx, int batch, size_t* bytes) {
  if (!ctx || !bytes) return fail(JAGG_EINVAL, "dit_workspace_bytes: null argument");
  if (batch < 1 || batch > MAX_BATCH) return fail(JAGG_EINVAL, "dit_workspace_bytes: batch must be 1..32");
  jg::Ws W;
  *bytes = jg::plan_ws(ctx->m, batch, nullptr, W);
  return JAGG_OK;
}

jagg_status jagg_ctx_set_workspace(jagg_ctx* ctx, void* ws, size_t bytes) {
  if (!ctx) return fail(JAGG_EINVAL, "jagg_ctx_set_workspace: null context");
  if ((uintptr_t)ws % 256) return fail(JAGG_EINVAL, "jagg_ctx_set_workspace: workspace must be 256-byte aligned");
  ctx->ws = ws;
  ctx->ws_bytes = ws ? bytes : 0;
  return JAGG_OK;
}

jagg_status dit_forward_save(jagg_ctx* ctx, const void* theta, const void* z, const float* t, const void* txt,
                             void* v_out, void* saved, int batch) {
  if (!ctx || !theta || !z || !t || !v_out) return fail(JAGG_EINVAL, "dit_forward_save: null argument");
  if (!ctx->m.c.block_only && !txt) return fail(JAGG_EINVAL, "dit_forward_save: txt is required");
  if (batch < 1 || batch > MAX_BATCH) return fail(JAGG_EINVAL, "dit_forward_save: batch must be 1..32");
  if (((uintptr_t)theta | (uintptr_t)z | (uintptr_t)v_out | (uintptr_t)saved | (uintptr_t)txt) % 16)
    return fail(JAGG_EINVAL, "dit_forward_save: device pointers must be 16-byte aligned");
  jagg_status st = need_ws(ctx, batch);
  if (st) return st;
  return to_status(jg::forward(ctx, theta, z, t, txt, v_out, saved, batch));
}

jagg_status dit_vjp(jagg_ctx* ctx, const void* theta, const void* saved, int batch, const void* s, void* dtheta,
                    float beta) {
  if (!ctx || !theta || !saved || !s || !dtheta) return fail(JAGG_EINVAL, "dit_vjp: null argument");
  if (batch < 1 || batch > MAX_BATCH) return fail(JAGG_EINVAL, "dit_vjp: batch must be 1..32");
  if (beta != 0.f && beta != 1.f) return fail(JAGG_EINVAL, "dit_vjp: beta must be 0 or 1");
  if (((uintptr_t)theta | (uintptr_t)saved | (uintptr_t)s | (uintptr_t)dtheta) % 16)
    return fail(JAGG_EINVAL, "dit_vjp: device pointers must be 16-byte aligned");
  jagg_status st = need_ws(ctx, batch);
  if (st) return st;
  return to_status(jg::vjp(ctx, theta, saved, batch, s, dtheta, beta));
}

jagg_status jagg_alpha(const float* t, int W, float* alpha_out) {
  if (!t || !alpha_out) return fail(JAGG_EINVAL, "jagg_alpha: null argument");
  if (W < 2) return fail(JAGG_EINVAL, "jagg_alpha: W must be >= 2");
  if (!decreasing(t, W)) return fail(JAGG_EINVAL, "jagg_alpha: t must be strictly decreasing");
  const double t0 = t[0], den = (double)t[0] - (double)t[W - 1];
  for (int j = 0; j < W; ++j) alpha_out[j] = (float)((t0 - (double)t[j]) / den);
  return JAGG_OK;
}

static jagg_status agg_weights(const float* t, int W, jg::AggArgs& a) {
  if (W < 2 || W > 64) return fail(JAGG_EINVAL, "aggregation: W must be 2..64");
  if (!decreasing(t, W)) return fail(JAGG_EINVAL, "aggregation: t must be strictly decreasing");
  const double t0 = t[0], den = (double)t[0] - (double)t[W - 1];
  for (int j = 0; j < W; ++j) {
    const double al = (t0 - (double)t[j]) / den;
    a.wb[j] = (float)(1.0 - al);
    a.wc[j] = (float)al;
  }
  a.W = W;
  return JAGG_OK;
}

jagg_status jagg_aggregate(jagg_ctx* ctx, const void* const* s, const float* t, int W, size_t n, int dtype,
                           void* s_base, void* s_corr) {
  if (!ctx || !s || !t || !s_base || !s_corr) return fail(JAGG_EINVAL, "jagg_aggregate: null argument");
  if (dtype != JAGG_F32 && dtype != JAGG_BF16) return fail(JAGG_EINVAL, "jagg_aggregate: unknown dtype");
  jg::AggArgs a;
  std::memset(&a, 0, sizeof(a));
  jagg_status st = agg_weights(t, W, a);
  if (st) return st;
  for (int j = 0; j < W; ++j) {
    if (!s[j]) return fail(JAGG_EINVAL, "jagg_aggregate: null s_j");
    a.s[j] = s[j];
  }
  a.n = n;
  a.split = n;
  a.base0 = a.base1 = s_base;
  a.corr0 = a.corr1 = s_corr;
  a.in_dt = a.out_dt = dtype;
  return to_status(jg::aggregate(a, ctx->stream));
}

jagg_status jagg_group_scores(jagg_ctx* ctx, const void* const* h, size_t n, int W, int dtype, double* score_out) {
  if (!ctx || !h || !score_out) return fail(JAGG_EINVAL, "jagg_group_scores: null argument");
  if (W < 2 || W > 8) return fail(JAGG_EINVAL, "jagg_group_scores: W must be 2..8");
  if (n == 0) return fail(JAGG_EINVAL, "jagg_group_scores: empty vectors");
  if (dtype != JAGG_F32 && dtype != JAGG_BF16) return fail(JAGG_EINVAL, "jagg_group_scores: unknown dtype");
  jg::Ws W0;
  jagg_status st = need_head_ws(ctx, W0, "jagg_group_scores");
  if (st) return st;
  jg::ScoreArgs a;
  std::memset(&a, 0, sizeof(a));
  for (int j = 0; j < W; ++j) {
    if (!h[j]) return fail(JAGG_EINVAL, "jagg_group_scores: null h_j");
    a.h[j] = h[j];
  }
  a.W = W;
  a.n = n;
  a.dt = dtype;
  int rc = jg::group_scores(a, W0.spart, W0.score, ctx->stream);
  if (rc) return (jagg_status)rc;
  if (hipMemcpyAsync(score_out, W0.score, sizeof(double), hipMemcpyDeviceToHost, ctx->stream) != hipSuccess ||
      hipStreamSynchronize(ctx->stream) != hipSuccess)
    return fail(JAGG_EDEVICE, "jagg_group_scores: copy of the score failed");
  return JAGG_OK;
}

}  // extern "C"

// ------------------------------------------------ allocation-free scoring
// Device scratch of jagg_group_scores_noalloc: the score pass's per-block fp64
// partial sums (SC_BLOCKS blocks x W(W+1)/2 pair products; 147,456 bytes at
// the largest W, 8).  Each device holds its own copy until the process ends.
// In host code `scratch` names a host-side stand-in, never the device memory:
// kernels get the address hipGetSymbolAddress returns for the current device.
static constexpr size_t NOALLOC_SCRATCH_BYTES = 147456;
static __device__ __align__(256) unsigned char scratch[NOALLOC_SCRATCH_BYTES];

namespace {
std::mutex g_scratch_mu;
void* g_scratch_dev[64] = {};

// The current device's copy of `scratch`, looked up on the first call made on
// that device and kept for the later ones.
jagg_status scratch_ptr(void** out, const char* who) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
    return fail(JAGG_EDEVICE, std::string(who) + ": no current device");
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(JAGG_EDEVICE, std::string(who) + ": address of the static scratch: " + hipGetErrorString(e));
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return JAGG_OK;
}
}  // namespace

extern "C" {

jagg_status jagg_group_scores_noalloc(jagg_ctx* ctx, const void* const* h, size_t n, int W, int dtype,
                                      double* score_dev) {
  const char* f = "jagg_group_scores_noalloc";
  if (!ctx || !h || !score_dev) return fail(JAGG_EINVAL, std::string(f) + ": null argument");
  if (W < 2 || W > 8) return fail(JAGG_EINVAL, std::string(f) + ": W must be 2..8");
  if (n == 0) return fail(JAGG_EINVAL, std::string(f) + ": empty vectors");
  if (dtype != JAGG_F32 && dtype != JAGG_BF16) return fail(JAGG_EINVAL, std::string(f) + ": unknown dtype");
  if ((uintptr_t)score_dev % 8) return fail(JAGG_EINVAL, std::string(f) + ": score_dev must be 8-byte aligned");
  const size_t need = jg::score_part_doubles(W) * sizeof(double);
  if (need > NOALLOC_SCRATCH_BYTES)
    return fail(JAGG_EINVAL, std::string(f) + ": W = " + std::to_string(W) + " needs " + std::to_string(need) +
                                 " bytes of scratch, more than the static " + std::to_string(NOALLOC_SCRATCH_BYTES));
  jg::ScoreArgs a;
  std::memset(&a, 0, sizeof(a));
  for (int j = 0; j < W; ++j) {
    if (!h[j]) return fail(JAGG_EINVAL, std::string(f) + ": null h_j");
    a.h[j] = h[j];
  }
  a.W = W;
  a.n = n;
  a.dt = dtype;
  void* part = nullptr;
  jagg_status st = scratch_ptr(&part, f);
  if (st) return st;
  // pass 1 writes every partial it reads back, so nothing needs clearing
  return to_status(jg::group_scores(a, (double*)part, score_dev, ctx->stream));
}

jagg_status jagg_route(const double* scores, int n_groups, double tau, double frac, unsigned char* use_jagg_out,
                       double* frac_out) {
  if (!use_jagg_out || n_groups <= 0) return fail(JAGG_EINVAL, "jagg_route: bad arguments");
  int n = 0;
  if (frac >= 0.0) {
    if (frac > 1.0) return fail(JAGG_EINVAL, "jagg_route: frac must lie in [0, 1]");
    n = (int)std::floor(frac * n_groups + 1e-6);
  } else {
    if (!scores) return fail(JAGG_EINVAL, "jagg_route: scores required when frac < 0");
    while (n < n_groups && scores[n] >= tau) ++n;
  }
  for (int g = 0; g < n_groups; ++g) use_jagg_out[g] = g < n ? 1 : 0;
  if (frac_out) *frac_out = (double)n / n_groups;
  return JAGG_OK;
}

jagg_status jagg_linear_grad(jagg_ctx* ctx, int kind, const void* dY, const void* other, const void* pre, int rows,
                             int n_out, int n_in, void* result, int result_dtype, float beta) {
  if (!ctx || !dY || !other || !result) return fail(JAGG_EINVAL, "jagg_linear_grad: null argument");
  if (kind != JAGG_DGRAD && kind != JAGG_DGRAD_GELU && kind != JAGG_WGRAD)
    return fail(JAGG_EINVAL, "jagg_linear_grad: unknown kind");
  if (rows < 1 || n_out < 1 || n_in < 1) return fail(JAGG_EINVAL, "jagg_linear_grad: sizes must be >= 1");
  if (result_dtype != JAGG_F32 && result_dtype != JAGG_BF16)
    return fail(JAGG_EINVAL, "jagg_linear_grad: unknown result dtype");
  if (kind == JAGG_DGRAD_GELU && (!pre || result_dtype != JAGG_BF16))
    return fail(JAGG_EINVAL, "jagg_linear_grad: the GELU kind needs pre and a bf16 result");
  if ((kind == JAGG_WGRAD ? (beta != 0.f && beta != 1.f) : beta != 0.f))
    return fail(JAGG_EINVAL, "jagg_linear_grad: beta must be 0 (or 1 for the weight gradient)");
  if (((uintptr_t)dY | (uintptr_t)other | (uintptr_t)pre | (uintptr_t)result) % 16)
    return fail(JAGG_EINVAL, "jagg_linear_grad: device pointers must be 16-byte aligned");
  jg::GemmArgs g;
  g.A = dY; g.a_dt = jg::BF16;
  g.B = other; g.b_dt = jg::BF16; g.tb = 1;
  g.epi.C = result; g.epi.c_dt = result_dtype;
  if (kind == JAGG_WGRAD) {
    g.lda = n_out; g.ta = 1;
    g.ldb = n_in;
    g.M = n_out; g.N = n_in; g.K = rows;
    g.epi.ldc = n_in; g.epi.beta = beta;
  } else {
    g.lda = n_out; g.ta = 0;
    g.ldb = n_in;
    g.M = rows; g.N = n_in; g.K = n_out;
    g.epi.ldc = n_in;
    if (kind == JAGG_DGRAD_GELU) {
      g.epi.mode = jg::EPI_GELU_BWD; g.epi.aux = (void*)pre; g.epi.ldaux = n_in; g.epi.aux_dt = jg::BF16;
    }
  }
  return to_status(jg::gemm(g, ctx->stream));
}

jagg_status jagg_group_backward(jagg_ctx* ctx, const void* theta, const void* saved_pair, int batch,
                                const void* const* s, const float* t, int W, void* dtheta, float beta) {
  if (!ctx || !theta || !saved_pair || !s || !t || !dtheta) return fail(JAGG_EINVAL, "jagg_group_backward: null argument");
  if (batch < 1 || 2 * batch > MAX_BATCH) return fail(JAGG_EINVAL, "jagg_group_backward: batch must be 1..16");
  if (beta != 0.f && beta != 1.f) return fail(JAGG_EINVAL, "jagg_group_backward: beta must be 0 or 1");
  const int B2 = 2 * batch;
  jagg_status st = need_ws(ctx, B2);
  if (st) return st;
  const jg::Model& m = ctx->m;
  jg::AggArgs a;
  std::memset(&a, 0, sizeof(a));
  st = agg_weights(t, W, a);
  if (st) return st;
  for (int j = 0; j < W; ++j) {
    if (!s[j] || (uintptr_t)s[j] % 16) return fail(JAGG_EINVAL, "jagg_group_backward: null or unaligned s_j");
    a.s[j] = s[j];
  }
  jg::Ws Wp;
  jg::plan_ws(m, B2, ctx->ws, Wp);
  const size_t es = jg::dsize(m.act);
  char* cot = (char*)Wp.cot;
  a.n = (size_t)batch * jg::out_elems(m);
  if (m.c.block_only) {
    const size_t txt = (size_t)batch * m.nt * m.D, img = (size_t)batch * m.ni * m.D;
    a.split = txt;
    a.base0 = cot;
    a.corr0 = cot + txt * es;
    a.base1 = cot + 2 * txt * es;
    a.corr1 = cot + (2 * txt + img) * es;
  } else {
    a.split = a.n;
    a.base0 = a.base1 = cot;
    a.corr0 = a.corr1 = cot + a.n * es;
  }
  a.in_dt = a.out_dt = m.act;
  int rc = jg::aggregate(a, ctx->stream);
  if (rc) return (jagg_status)rc;
  return to_status(jg::vjp(ctx, theta, saved_pair, B2, cot, dtheta, beta));
}

jagg_status jagg_endpoint_backward(jagg_ctx* ctx, const void* theta, const void* saved, int batch, const void* const* s,
                                   const float* t, int W, int endpoint, void* dtheta, float beta) {
  if (!ctx || !theta || !saved || !s || !t || !dtheta) return fail(JAGG_EINVAL, "jagg_endpoint_backward: null argument");
  if (batch < 1 || batch > MAX_BATCH) return fail(JAGG_EINVAL, "jagg_endpoint_backward: batch must be 1..32");
  if (endpoint != 0 && endpoint != 1) return fail(JAGG_EINVAL, "jagg_endpoint_backward: endpoint must be 0 or 1");
  if (beta != 0.f && beta != 1.f) return fail(JAGG_EINVAL, "jagg_endpoint_backward: beta must be 0 or 1");
  if (((uintptr_t)theta | (uintptr_t)saved | (uintptr_t)dtheta) % 16)
    return fail(JAGG_EINVAL, "jagg_endpoint_backward: device pointers must be 16-byte aligned");
  jagg_status st = need_ws(ctx, batch);
  if (st) return st;
  jg::AggArgs a;
  std::memset(&a, 0, sizeof(a));
  st = agg_weights(t, W, a);
  if (st) return st;
  for (int j = 0; j < W; ++j) {
    if (!s[j] || (uintptr_t)s[j] % 16) return fail(JAGG_EINVAL, "jagg_endpoint_backward: null or unaligned s_j");
    a.s[j] = s[j];
  }
  const jg::Model& m = ctx->m;
  jg::Ws Wb;
  jg::plan_ws(m, batch, ctx->ws, Wb);
  // the composite of this endpoint only, in the batch-B output layout
  a.n = (size_t)batch * jg::out_elems(m);
  a.split = a.n;
  if (endpoint == 0) a.base0 = a.base1 = Wb.cot;
  else a.corr0 = a.corr1 = Wb.cot;
  a.in_dt = a.out_dt = m.act;
  int rc = jg::aggregate(a, ctx->stream);
  if (rc) return (jagg_status)rc;
  return to_status(jg::vjp(ctx, theta, saved, batch, Wb.cot, dtheta, beta));
}

jagg_status jagg_grad_compare(jagg_ctx* ctx, const void* a, const void* b, size_t n, int dtype, double* out) {
  if (!ctx || !a || !b || !out) return fail(JAGG_EINVAL, "jagg_grad_compare: null argument");
  if (n == 0) return fail(JAGG_EINVAL, "jagg_grad_compare: empty vectors");
  if (dtype != JAGG_F32 && dtype != JAGG_BF16) return fail(JAGG_EINVAL, "jagg_grad_compare: unknown dtype");
  if (((uintptr_t)a | (uintptr_t)b) % 16) return fail(JAGG_EINVAL, "jagg_grad_compare: vectors must be 16-byte aligned");
  jg::Ws W0;
  jagg_status st = need_head_ws(ctx, W0, "jagg_grad_compare");
  if (st) return st;
  int rc = jg::grad_compare(a, b, n, dtype, W0.spart, W0.score, ctx->stream);
  if (rc) return (jagg_status)rc;
  if (hipMemcpyAsync(out, W0.score, 3 * sizeof(double), hipMemcpyDeviceToHost, ctx->stream) != hipSuccess ||
      hipStreamSynchronize(ctx->stream) != hipSuccess)
    return fail(JAGG_EDEVICE, "jagg_grad_compare: copy of the sums failed");
  quality_from_sums(out);
  return JAGG_OK;
}

jagg_status jagg_count_nonfinite(jagg_ctx* ctx, const void* x, size_t n, int dtype, unsigned long long* count) {
  if (!ctx || !x || !count) return fail(JAGG_EINVAL, "jagg_count_nonfinite: null argument");
  if (n == 0) return fail(JAGG_EINVAL, "jagg_count_nonfinite: empty vector");
  if (dtype != JAGG_F32 && dtype != JAGG_BF16) return fail(JAGG_EINVAL, "jagg_count_nonfinite: unknown dtype");
  if ((uintptr_t)x % 16) return fail(JAGG_EINVAL, "jagg_count_nonfinite: vector must be 16-byte aligned");
  jg::Ws W0;
  jagg_status st = need_head_ws(ctx, W0, "jagg_count_nonfinite");
  if (st) return st;
  auto* part = (unsigned long long*)W0.spart;
  auto* slot = (unsigned long long*)W0.score;
  int rc = jg::count_nonfinite(x, n, dtype, part, slot, ctx->stream);
  if (rc) return (jagg_status)rc;
  if (hipMemcpyAsync(count, slot, sizeof(unsigned long long), hipMemcpyDeviceToHost, ctx->stream) != hipSuccess ||
      hipStreamSynchronize(ctx->stream) != hipSuccess)
    return fail(JAGG_EDEVICE, "jagg_count_nonfinite: copy of the count failed");
  return JAGG_OK;
}

jagg_status jagg_window_quality(jagg_ctx* ctx, const void* theta, const void* saved_pair,
                                const void* const* saved_steps, int batch, const void* const* s, const float* t, int W,
                                void* g_jagg, void* g_exact, void* g_ablate, double* out) {
  const char* f = "jagg_window_quality";
  if (!ctx || !theta || !saved_pair || !saved_steps || !s || !t || !g_jagg || !g_exact || !g_ablate || !out)
    return fail(JAGG_EINVAL, std::string(f) + ": null argument");
  if (W < 2 || W > 64) return fail(JAGG_EINVAL, std::string(f) + ": W must be 2..64");
  if (((uintptr_t)g_jagg | (uintptr_t)g_exact | (uintptr_t)g_ablate) % 16)
    return fail(JAGG_EINVAL, std::string(f) + ": gradient buffers must be 16-byte aligned");
  for (int j = 0; j < W; ++j)
    if (!saved_steps[j] || !s[j]) return fail(JAGG_EINVAL, std::string(f) + ": null saved_j or s_j");
  if (!decreasing(t, W)) return fail(JAGG_EINVAL, std::string(f) + ": t must be strictly decreasing");
  jg::Ws W0;
  jagg_status st = need_head_ws(ctx, W0, f);
  if (st) return st;
  const int gdt = ctx->m.grad;
  const size_t n = ctx->m.total;
  // the three group gradients of the window
  st = jagg_group_backward(ctx, theta, saved_pair, batch, s, t, W, g_jagg, 0.f);
  if (st) return st;
  st = perstep_group_backward(ctx, theta, saved_steps, batch, s, W, g_exact, 0.f);
  if (st) return st;
  // ablation: the endpoint signals alone, weight one each (alpha = (0, 1))
  const void* s2[2] = {s[0], s[W - 1]};
  const float t2[2] = {t[0], t[W - 1]};
  st = jagg_group_backward(ctx, theta, saved_pair, batch, s2, t2, 2, g_ablate, 0.f);
  if (st) return st;
  double q[5];
  st = jagg_grad_compare(ctx, g_jagg, g_exact, n, gdt, q);
  if (st) return st;
  out[0] = q[3];
  out[1] = q[4];
  st = jagg_grad_compare(ctx, g_ablate, g_exact, n, gdt, q);
  if (st) return st;
  out[2] = q[3];
  out[3] = q[4];
  return JAGG_OK;
}

// Validates one GRPO window and fills the arguments shared by the three
// GRPO entry points (everything but the outputs).
static jagg_status grpo_args(const jagg_ctx* ctx, const jagg_grpo_window* w, int batch, jg::GrpoArgs& a,
                             const char* who) {
  const std::string f = who;
  if (!w || !w->v_hat || !w->z || !w->t || !w->sigma || !w->logp_old || !w->adv)
    return fail(JAGG_EINVAL, f + ": null argument");
  if (batch < 1 || batch > 16) return fail(JAGG_EINVAL, f + ": batch must be 1..16");
  const int W = w->W;
  if (W < 2 || W > jg::GRPO_MAX_W) return fail(JAGG_EINVAL, f + ": W must be 2..16");
  if (!(w->clip_eps >= 0.f) || !(w->adv_clip > 0.f)) return fail(JAGG_EINVAL, f + ": bad clip range or advantage clamp");
  std::memset(&a, 0, sizeof(a));
  if (!decreasing(w->t, W + 1)) return fail(JAGG_EINVAL, f + ": t_0 .. t_W must be strictly decreasing");
  const double t0 = w->t[0], den = (double)w->t[0] - (double)w->t[W - 1];
  for (int j = 0; j < W; ++j) {
    if (!(w->sigma[j] > 0.f)) return fail(JAGG_EINVAL, f + ": sigma_j must be positive");
    if (!w->v_hat[j] || (uintptr_t)w->v_hat[j] % 16) return fail(JAGG_EINVAL, f + ": null or unaligned v_j");
    const double al = (t0 - (double)w->t[j]) / den;
    a.wb[j] = (float)(1.0 - al);
    a.wc[j] = (float)al;
    a.dts[j] = (double)w->t[j + 1] - (double)w->t[j];
    a.sigma[j] = w->sigma[j];
    a.v[j] = w->v_hat[j];
    a.vb[j] = w->v_batch ? w->v_batch[j] : batch;
    a.vk[j] = w->v_index ? w->v_index[j] : 0;
    if (a.vk[j] < 0 || a.vb[j] < batch || a.vk[j] + batch > a.vb[j] || a.vb[j] > 64)
      return fail(JAGG_EINVAL, f + ": v_batch / v_index out of range");
  }
  for (int j = 0; j <= W; ++j) {
    if (!w->z[j] || (uintptr_t)w->z[j] % 16) return fail(JAGG_EINVAL, f + ": null or unaligned z_j");
    a.z[j] = w->z[j];
  }
  const jg::Model& m = ctx->m;
  a.W = W;
  a.B = batch;
  a.dt = m.act;
  if (m.c.block_only) {  // stream-major rows: text rows of all samples, then image rows
    a.len0 = (size_t)m.nt * m.D;
    a.len1 = (size_t)m.ni * m.D;
    a.split = (size_t)batch * a.len0;
  } else {
    a.len0 = 0;
    a.len1 = jg::out_elems(m);
    a.split = 0;
  }
  a.n = (size_t)batch * (a.len0 + a.len1);
  a.logp_old = w->logp_old;
  a.adv = w->adv;
  a.eps = w->clip_eps;
  a.adv_clip = w->adv_clip;
  return JAGG_OK;
}

static jagg_status grpo_run(jagg_ctx* ctx, jg::GrpoArgs& a, double* stats) {
  jg::Ws W0;
  jagg_status st = need_head_ws(ctx, W0, "GRPO window");
  if (st) return st;
  return to_status(jg::grpo_window(a, W0.spart, W0.gcoef, stats, ctx->stream));
}

jagg_status jagg_grpo_composites(jagg_ctx* ctx, const jagg_grpo_window* w, int batch, void* s_base, void* s_corr,
                                 double* stats) {
  if (!ctx || !s_base || !s_corr) return fail(JAGG_EINVAL, "jagg_grpo_composites: null argument");
  if (((uintptr_t)s_base | (uintptr_t)s_corr) % 16) return fail(JAGG_EINVAL, "jagg_grpo_composites: unaligned output");
  jg::GrpoArgs a;
  jagg_status st = grpo_args(ctx, w, batch, a, "jagg_grpo_composites");
  if (st) return st;
  a.mode = 0;
  a.osplit = a.n;
  a.base0 = a.base1 = s_base;
  a.corr0 = a.corr1 = s_corr;
  return grpo_run(ctx, a, stats);
}

jagg_status jagg_grpo_upstream(jagg_ctx* ctx, const jagg_grpo_window* w, int batch, void* const* s_out,
                               double* stats) {
  if (!ctx || !s_out) return fail(JAGG_EINVAL, "jagg_grpo_upstream: null argument");
  jg::GrpoArgs a;
  jagg_status st = grpo_args(ctx, w, batch, a, "jagg_grpo_upstream");
  if (st) return st;
  for (int j = 0; j < a.W; ++j) {
    if (!s_out[j] || (uintptr_t)s_out[j] % 16) return fail(JAGG_EINVAL, "jagg_grpo_upstream: null or unaligned s_j");
    a.s_out[j] = s_out[j];
  }
  a.mode = 1;
  return grpo_run(ctx, a, stats);
}

jagg_status jagg_grpo_group_backward(jagg_ctx* ctx, const void* theta, const void* saved_pair, int batch,
                                     const jagg_grpo_window* w, void* dtheta, float beta, double* stats) {
  if (!ctx || !theta || !saved_pair || !dtheta) return fail(JAGG_EINVAL, "jagg_grpo_group_backward: null argument");
  if (beta != 0.f && beta != 1.f) return fail(JAGG_EINVAL, "jagg_grpo_group_backward: beta must be 0 or 1");
  jg::GrpoArgs a;
  jagg_status st = grpo_args(ctx, w, batch, a, "jagg_grpo_group_backward");
  if (st) return st;
  const int B2 = 2 * batch;
  st = need_ws(ctx, B2);
  if (st) return st;
  const jg::Model& m = ctx->m;
  jg::Ws Wp;
  jg::plan_ws(m, B2, ctx->ws, Wp);
  const size_t es = jg::dsize(m.act);
  char* cot = (char*)Wp.cot;
  // composites straight into the cotangent of the batch-2B endpoint pair
  a.mode = 0;
  if (m.c.block_only) {
    const size_t txt = (size_t)batch * m.nt * m.D, img = (size_t)batch * m.ni * m.D;
    a.osplit = txt;
    a.base0 = cot;
    a.corr0 = cot + txt * es;
    a.base1 = cot + 2 * txt * es;
    a.corr1 = cot + (2 * txt + img) * es;
  } else {
    a.osplit = a.n;
    a.base0 = a.base1 = cot;
    a.corr0 = a.corr1 = cot + a.n * es;
  }
  st = grpo_run(ctx, a, stats);
  if (st) return st;
  return to_status(jg::vjp(ctx, theta, saved_pair, B2, cot, dtheta, beta));
}

jagg_status perstep_group_backward(jagg_ctx* ctx, const void* theta, const void* const* saved, int batch,
                                   const void* const* s, int W, void* dtheta, float beta) {
  if (!ctx || !theta || !saved || !s || !dtheta) return fail(JAGG_EINVAL, "perstep_group_backward: null argument");
  if (W < 1 || W > 64) return fail(JAGG_EINVAL, "perstep_group_backward: W must be 1..64");
  for (int j = 0; j < W; ++j)
    if (!saved[j] || !s[j]) return fail(JAGG_EINVAL, "perstep_group_backward: null saved_j or s_j");
  for (int j = 0; j < W; ++j) {
    jagg_status st = dit_vjp(ctx, theta, saved[j], batch, s[j], dtheta, j == 0 ? beta : 1.f);
    if (st) return st;
  }
  return JAGG_OK;
}

jagg_status jagg_trajectory_backward(jagg_ctx* ctx, const void* theta, int T, int W, int batch,
                                     const void* const* saved_pairs, const void* const* saved_steps,
                                     const void* const* s, const float* t, const unsigned char* use_jagg,
                                     void* dtheta, float beta) {
  const char* f = "jagg_trajectory_backward";
  if (!ctx || !theta || !s || !t || !dtheta) return fail(JAGG_EINVAL, std::string(f) + ": null argument");
  if (W < 2 || W > 64 || T < 1) return fail(JAGG_EINVAL, std::string(f) + ": need 2 <= W <= 64 and T >= 1");
  if (beta != 0.f && beta != 1.f) return fail(JAGG_EINVAL, std::string(f) + ": beta must be 0 or 1");
  if (!decreasing(t, T)) return fail(JAGG_EINVAL, std::string(f) + ": t must be strictly decreasing");
  const int n_full = T / W;
  if (n_full > 0 && !use_jagg) return fail(JAGG_EINVAL, std::string(f) + ": use_jagg is required");
  bool any_jagg = false;
  // every pointer a pass will read, checked before the first launch
  for (int g = 0; g <= n_full; ++g) {
    const int k0 = g * W, k1 = g < n_full ? k0 + W : T;
    if (k0 >= k1) continue;
    const bool j = g < n_full && use_jagg[g] == 1;
    if (g < n_full && use_jagg[g] > 1) return fail(JAGG_EINVAL, std::string(f) + ": use_jagg entries must be 0 or 1");
    if (j) {
      if (!saved_pairs || !saved_pairs[g]) return fail(JAGG_EINVAL, std::string(f) + ": null saved pair of a JAGG window");
      if (batch < 1 || 2 * batch > MAX_BATCH) return fail(JAGG_EINVAL, std::string(f) + ": batch must be 1..16");
      any_jagg = true;
    }
    for (int k = k0; k < k1; ++k) {
      if (!s[k] || (uintptr_t)s[k] % 16) return fail(JAGG_EINVAL, std::string(f) + ": null or unaligned s_k");
      if (!j && (!saved_steps || !saved_steps[k]))
        return fail(JAGG_EINVAL, std::string(f) + ": null saved forward of a per-step step");
    }
  }
  if (batch < 1 || batch > MAX_BATCH) return fail(JAGG_EINVAL, std::string(f) + ": batch must be 1..32");
  jagg_status st = need_ws(ctx, any_jagg ? 2 * batch : batch);
  if (st) return st;
  float b = beta;
  for (int g = 0; g <= n_full; ++g) {
    const int k0 = g * W, k1 = g < n_full ? k0 + W : T;
    if (k0 >= k1) continue;
    if (g < n_full && use_jagg[g])
      st = jagg_group_backward(ctx, theta, saved_pairs[g], batch, s + k0, t + k0, W, dtheta, b);
    else
      st = perstep_group_backward(ctx, theta, saved_steps + k0, batch, s + k0, k1 - k0, dtheta, b);
    if (st) return st;
    b = 1.f;
  }
  return JAGG_OK;
}

}  // extern "C"
