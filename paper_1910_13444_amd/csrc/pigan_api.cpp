// Host side of libpigan.so: argument checks, workspace planning, the chunked
// orchestration of one PI-GAN training step and the C entry points declared
// in include/pigan.h.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"
#include "pointwise.h"
#include "optim.h"

namespace pigan {

// ---------------------------------------------------------------------------
// errors
// ---------------------------------------------------------------------------
static thread_local std::string g_err;

static pigan_status fail(pigan_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define HIP_TRY(expr)                                                                       \
  do {                                                                                      \
    hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess) return fail(PIGAN_EDEVICE, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

// ---------------------------------------------------------------------------
// kernel timing record (enabled by pigan_profile_enable)
// ---------------------------------------------------------------------------
struct ProfRec {
  std::string name;
  hipEvent_t a, b;
  double flops, bytes;
};
static std::mutex g_pm;
static bool g_prof = false;
static std::vector<ProfRec> g_recs;
static std::vector<hipEvent_t> g_pool;

static hipEvent_t pool_get() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void prof_begin(hipStream_t st, const char* name, double flops, double bytes) {
  std::lock_guard<std::mutex> lk(g_pm);
  if (!g_prof) return;
  ProfRec r{name, pool_get(), pool_get(), flops, bytes};
  if (r.a) (void)hipEventRecord(r.a, st);
  g_recs.push_back(r);
}

void prof_end(hipStream_t st) {
  std::lock_guard<std::mutex> lk(g_pm);
  if (!g_prof || g_recs.empty()) return;
  if (g_recs.back().b) (void)hipEventRecord(g_recs.back().b, st);
}

struct ProfScope {
  hipStream_t st;
  ProfScope(hipStream_t s, const char* name, double flops, double bytes) : st(s) {
    prof_begin(s, name, flops, bytes);
  }
  ~ProfScope() { prof_end(st); }
};

// ---------------------------------------------------------------------------
// shapes and workspace carving
// ---------------------------------------------------------------------------
static inline int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

struct Carver {
  size_t off = 0;
  size_t take(size_t bytes) {
    off = (size_t)round_up((int64_t)off, 256);
    const size_t o = off;
    off += bytes;
    return o;
  }
};

static size_t esize(int32_t dt) { return dt == PIGAN_FP32 ? 4 : 2; }

struct MlpOff {  // offsets (in floats) of one group's packed parameters
  int in_dim, L, W;
  int64_t n;
  std::vector<int64_t> w, b;
  int64_t wout;      // output layer: heads x [w (W), b]
  void init(int in_dim_, int L_, int W_, int heads = 1) {
    in_dim = in_dim_;
    L = L_;
    W = W_;
    w.assign(L + 1, 0);
    b.assign(L + 1, 0);
    int64_t off = 0;
    int fan = in_dim;
    for (int l = 1; l <= L; ++l) {
      w[l] = off;
      off += (int64_t)W * fan;
      b[l] = off;
      off += W;
      fan = W;
    }
    wout = off;
    n = off + (int64_t)heads * (W + 1);
  }
};

// layer l (1-based) of a shared trunk ends a residual block: h_l = tanh(a_l) + h_{l-2}
static bool trunk_skip(int l) { return l >= 3 && l % 2 == 1; }

static bool width_ok(int W) {
  if (W < 32 || W > 4096 || W % 32) return false;
  return W <= 256 ? (256 % W == 0) : (W % 256 == 0);
}

static pigan_status check_mlp(const pigan_mlp* m, const char* what) {
  if (!m) return fail(PIGAN_EINVAL, "%s: null shape", what);
  if (m->n_groups < 1 || m->n_groups > 65535) return fail(PIGAN_EINVAL, "%s: n_groups=%d out of [1,65535]", what, m->n_groups);
  if (m->in_dim < 1) return fail(PIGAN_EINVAL, "%s: in_dim=%d must be >= 1", what, m->in_dim);
  if (m->n_hidden < 1) return fail(PIGAN_EINVAL, "%s: n_hidden=%d must be >= 1", what, m->n_hidden);
  if (m->width < 1) return fail(PIGAN_EINVAL, "%s: width=%d must be >= 1", what, m->width);
  if (!width_ok(m->width))
    return fail(PIGAN_ENOTSUP, "%s: width=%d unsupported (multiple of 32 dividing 256, or multiple of 256 up to 4096)",
                what, m->width);
  return PIGAN_OK;
}

static pigan_status check_dtype(int32_t dt) {
  if (dt != PIGAN_FP32 && dt != PIGAN_BF16 && dt != PIGAN_FP16) return fail(PIGAN_EINVAL, "unknown dtype %d", (int)dt);
  return PIGAN_OK;
}

// row chunks per sample of the first-layer reverse pass: about 1024 blocks
static int first_bwd_chunks(int S) {
  int c = (1024 + S - 1) / S;
  return c < 1 ? 1 : (c > 64 ? 64 : c);
}

// points per block of the output-layer reverse pass: about 2048 blocks for
// widths >= 512 (a block then covers only one or two points per pass over
// its threads; eight blocks per CU keep enough loads in flight), 512 below
// (a block covers 16 points per pass; more blocks only add partials)
static int64_t ob_ppb(int64_t n_points, int W) {
  const int64_t blocks = W >= 512 ? 2048 : 512;
  int64_t p = (n_points + blocks - 1) / blocks;
  return p < 8 ? 8 : p;
}

// ---------------------------------------------------------------------------
// storage and product policy
// ---------------------------------------------------------------------------
// The collocation rows (value and derivative streams feeding the residual)
// are stored in the step's type T.  The adversarial path -- the generators'
// sensor rows, whose cotangents come from the critic, and the critic itself
// -- is stored in fp32 and multiplied with split products (ProdMode): at the
// initial weights a critic is far less sensitive to a uniform shift of a
// sensor block than to the single sensors it sums over, so the generators'
// gradients there are small differences of large per-row terms.  Rounding
// every row on that path to a 16-bit format, or accumulating its long
// contractions in fp32, moves them by several hundred rounding units.  In
// fp32 mode those products run on the fp64 matrix core (fp32 operands are
// exact in fp64, one rounding per result); in 16-bit modes two bf16 pieces
// per operand (about 16 significand bits each, three products) keep those
// gradients well inside the accuracy of the 16-bit collocation rows.
template <class T> constexpr int adv_pm() { return sizeof(T) == 2 ? PM_SPLIT2 : PM_F64; }
// split-K partials of these product modes are fp64
static bool pm_wide(int pm) { return pm == PM_SPLIT3 || pm == PM_F64; }
// 16-bit storage: the collocation forward products take two-term weights
// [W_hi | W_lo], so the generated fields and their derivatives see the fp32
// weights to about 16 significand bits (the residual at the initial weights is
// a small difference of jet products and amplifies a one-term rounding).
template <class T> constexpr bool two_term() { return sizeof(T) == 2; }

static const char* pm_tag(int pm) {
  return pm == PM_SPLIT2 ? "_x2" : (pm == PM_SPLIT3 ? "_x3" : (pm == PM_F64 ? "_f64" : ""));
}

// ---------------------------------------------------------------------------
// training-step plan
// ---------------------------------------------------------------------------
// One network's buffers for a chunk of samples.  Sensor rows (value stream
// only, fp32) and collocation stream rows (storage type T, stream k of point p
// at row k * n_col + p) have separate activation buffers; the output jets and
// their cotangents are fp32 vectors [sensor outputs | stream planes].
struct NetBuf {
  MlpOff off;
  int nd1 = 0, nd2 = 0, n_s = 0;
  int64_t n_sen = 0, n_col = 0;
  int64_t Rs = 0, Rc = 0;    // planned sensor rows / collocation stream rows per group
  int64_t R = 0;             // jet rows per group (Rs + Rc)
  int64_t rows = 0;          // jet rows used by the current chunk (<= R)
  std::vector<size_t> As, Hs, Ac, Hc;   // index 1..L
  size_t dAs[2] = {0, 0}, dAc[2] = {0, 0};
  // wc: collocation forward weights (two-term rows in 16-bit storage), wcT
  // their transposes (reverse pass); ws, wsT: fp32 copies and transposes for
  // the sensor rows (aligned rows: a packed parameter vector is only 4-byte
  // aligned per group)
  size_t jet = 0, gbar = 0, zp = 0, wc = 0, wcT = 0, ws = 0, wsT = 0, fb = 0, ob = 0;
  int64_t ob_slots = 0;
  int64_t ppb_sen = 8, ppb_col = 8;
  int nrc = 1;       // row chunks per sample in the first-layer reverse pass
  // shared trunk: residual blocks, a second head (u) with its own jets and
  // cotangents, the skip cotangent buffers, and the concatenated sensor
  // locations [Y sensors ; u sensors]
  bool skip = false;
  int heads = 1;
  size_t jet2 = 0, gbar2 = 0, ghs = 0, ghc = 0, xsc = 0;
  int C() const { return 1 + nd1 + nd2; }
};

// the critic: fp32 storage throughout
struct DiscBuf {
  MlpOff off;
  int Kp = 0;
  int64_t Bmax = 0;
  std::vector<size_t> A, H;
  size_t X0 = 0, dA[2] = {0, 0}, score = 0, seed = 0, w1 = 0, w1T = 0, wc = 0, wcT = 0, ob = 0;
  int64_t ob_slots = 0, ppb = 8;
};

struct StepPlan {
  bool trunk = false;   // one shared-trunk generator (in Y) instead of the Y / u pair
  int G = 1, Sc = 1;
  size_t es = 4;
  NetBuf Y, U;
  DiscBuf D;
  size_t dwp = 0, dwdb = 0, rpart = 0, acc = 0;
  size_t gpg = 0, gpp = 0;   // gradient penalty: critic input gradients [Sc x n_in] fp32, row terms [Sc] fp64
  // domain decomposition: residual and its critic cotangent [Sc*P] fp32, the
  // critics' fake-row input cotangents [D][Sc][Kp] fp32
  size_t hr = 0, hgn = 0, hdx = 0;
  int GD = 1;
  int64_t dwp_floats = 0, dwdb_floats = 0;
  int rblocks = 0;
  size_t total = 0;
};

static void plan_net(Carver& cv, NetBuf& nb, const pigan_mlp& m, int d, int nd2, int n_s, int Sc, int P, size_t es,
                     int G, bool trunk = false) {
  nb.skip = trunk;
  nb.heads = trunk ? 2 : 1;
  nb.off.init(m.in_dim, m.n_hidden, m.width, nb.heads);
  nb.nd1 = d;
  nb.nd2 = nd2;
  nb.n_s = n_s;
  nb.n_sen = (int64_t)Sc * n_s;
  nb.n_col = (int64_t)Sc * P;
  nb.Rs = nb.n_sen;
  nb.Rc = nb.C() * nb.n_col;
  nb.R = nb.Rs + nb.Rc;
  nb.rows = nb.R;
  const int L = m.n_hidden, W = m.width;
  const size_t act_s = (size_t)nb.Rs * W * 4 * G, act_c = (size_t)nb.Rc * W * es * G;
  nb.As.assign(L + 1, 0);
  nb.Hs.assign(L + 1, 0);
  nb.Ac.assign(L + 1, 0);
  nb.Hc.assign(L + 1, 0);
  for (int l = 1; l <= L; ++l) {
    nb.As[l] = cv.take(act_s);
    nb.Hs[l] = cv.take(act_s);
    nb.Ac[l] = cv.take(act_c);
    nb.Hc[l] = cv.take(act_c);
  }
  for (int i = 0; i < 2; ++i) {
    nb.dAs[i] = cv.take(act_s);
    nb.dAc[i] = cv.take(act_c);
  }
  nb.jet = cv.take((size_t)nb.R * 4 * G);
  nb.gbar = cv.take((size_t)nb.R * 4 * G);
  nb.zp = cv.take((size_t)Sc * W * 4 * G);
  const size_t nw = (size_t)std::max(L - 1, 1) * W * W * G;
  nb.wc = cv.take(nw * es * (es == 2 ? 2 : 1));
  nb.wcT = cv.take(nw * es);
  nb.ws = cv.take(nw * 4);
  nb.wsT = cv.take(nw * 4);
  nb.nrc = first_bwd_chunks(Sc);
  nb.fb = cv.take((size_t)Sc * nb.nrc * 7 * W * 8 * G);
  nb.ppb_sen = ob_ppb(nb.n_sen, W);
  nb.ppb_col = ob_ppb(nb.n_col, W);
  nb.ob_slots = out_bwd_blocks(nb.n_sen, (int)nb.ppb_sen) + out_bwd_blocks(nb.n_col, (int)nb.ppb_col);
  nb.ob = cv.take((size_t)nb.ob_slots * nb.heads * (W + 1) * 8 * G);
  if (trunk) {
    nb.jet2 = cv.take((size_t)nb.R * 4 * G);
    nb.gbar2 = cv.take((size_t)nb.R * 4 * G);
    if (L >= 3) {
      nb.ghs = cv.take(act_s);
      nb.ghc = cv.take(act_c);
    }
    nb.xsc = cv.take((size_t)n_s * d * 4 * G);
  }
}

static void plan_disc(Carver& cv, DiscBuf& D, const pigan_mlp& disc, int64_t Bmax, int GD) {
  D.off.init(disc.in_dim, disc.n_hidden, disc.width);
  const int WD = disc.width, LD = disc.n_hidden;
  D.Kp = (int)round_up(disc.in_dim, 32);
  D.Bmax = Bmax;
  D.X0 = cv.take((size_t)D.Bmax * D.Kp * 4 * GD);
  D.A.assign(LD + 1, 0);
  D.H.assign(LD + 1, 0);
  const size_t act = (size_t)D.Bmax * WD * 4 * GD;
  for (int l = 1; l <= LD; ++l) {
    D.A[l] = cv.take(act);
    D.H[l] = cv.take(act);
  }
  D.dA[0] = cv.take(act);
  D.dA[1] = cv.take(act);
  D.score = cv.take((size_t)D.Bmax * 4 * GD);
  D.seed = cv.take((size_t)D.Bmax * 4 * GD);
  D.w1 = cv.take((size_t)WD * D.Kp * 4 * GD);
  D.w1T = cv.take((size_t)WD * D.Kp * 4 * GD);
  D.wc = cv.take((size_t)std::max(LD - 1, 1) * WD * WD * 4 * GD);
  D.wcT = cv.take((size_t)std::max(LD - 1, 1) * WD * WD * 4 * GD);
  D.ppb = ob_ppb(D.Bmax, WD);
  D.ob_slots = out_bwd_blocks(D.Bmax, (int)D.ppb);
  D.ob = cv.take((size_t)D.ob_slots * (WD + 1) * 8 * GD);
}

// split-K partials (8 bytes per entry: fp32, or fp64 for PM_SPLIT3): the
// largest of all weight-gradient launches of a plan.  Gx groups per launch.
static void plan_partials(Carver& cv, StepPlan& pl, const pigan_step_desc* s, bool trunk, int Gg, int GD) {
  int64_t mx = 0, mxb = 0;
  auto consider = [&](int64_t R, int N, int J, int eb, int Gx) {
    int ns;
    int64_t rps;
    dw_split_plan(R, N, J, eb, Gx, &ns, &rps);
    mx = std::max(mx, (int64_t)ns * N * J * Gx);
    mxb = std::max(mxb, (int64_t)ns * N * Gx);
  };
  for (const NetBuf* nb : {&pl.Y, &pl.U}) {
    if (nb == &pl.U && trunk) continue;
    const int L = nb->off.L, W = nb->off.W;
    if (L > 1) {
      consider(nb->Rs, W, W, 4, Gg);
      consider(nb->Rc, W, W, (int)pl.es, Gg);
    }
  }
  const DiscBuf& D = pl.D;
  consider(D.Bmax, s->disc.width, D.Kp, 4, GD);
  if (s->disc.n_hidden > 1) consider(D.Bmax, s->disc.width, s->disc.width, 4, GD);
  pl.dwp_floats = mx;
  pl.dwdb_floats = mxb;
  pl.dwp = cv.take((size_t)mx * 8);
  pl.dwdb = cv.take((size_t)mxb * 8);
}

static void plan_step(const pigan_step_desc* s, int Sc, StepPlan& pl, bool trunk = false) {
  Carver cv;
  pl.trunk = trunk;
  pl.G = s->genY.n_groups;
  pl.Sc = Sc;
  pl.es = esize(s->dt);
  const int G = pl.G;
  if (trunk) {
    plan_net(cv, pl.Y, s->genY, s->d, s->d, s->n_sY + s->n_sU, Sc, s->P, pl.es, G, true);
  } else {
    plan_net(cv, pl.Y, s->genY, s->d, 0, s->n_sY, Sc, s->P, pl.es, G);
    plan_net(cv, pl.U, s->genU, s->d, s->d, s->n_sU, Sc, s->P, pl.es, G);
  }
  plan_disc(cv, pl.D, s->disc, (int64_t)Sc + s->B_r, G);
  plan_partials(cv, pl, s, trunk, G, G);
  pl.rblocks = residual_blocks((int64_t)Sc * s->P);
  pl.rpart = cv.take((size_t)pl.rblocks * 8 * G);
  pl.acc = cv.take((size_t)4 * 8 * G);
  if (s->lambda_gp > 0.0f) {
    pl.gpg = cv.take((size_t)Sc * s->disc.in_dim * 4 * G);
    pl.gpp = cv.take((size_t)Sc * 8 * G);
  }
  pl.total = round_up((int64_t)cv.off, 256);
}

// one generator (a pair, or the shared trunk in the Y slot; a single group)
// and s->disc.n_groups critics
static void plan_hier(const pigan_step_desc* s, int Sc, StepPlan& pl, bool trunk = false) {
  Carver cv;
  pl.trunk = trunk;
  pl.G = 1;
  pl.GD = s->disc.n_groups;
  pl.Sc = Sc;
  pl.es = esize(s->dt);
  const int GD = pl.GD;
  if (trunk) {
    plan_net(cv, pl.Y, s->genY, s->d, s->d, s->n_sY + s->n_sU, Sc, s->P, pl.es, 1, true);
  } else {
    plan_net(cv, pl.Y, s->genY, s->d, 0, s->n_sY, Sc, s->P, pl.es, 1);
    plan_net(cv, pl.U, s->genU, s->d, s->d, s->n_sU, Sc, s->P, pl.es, 1);
  }
  plan_disc(cv, pl.D, s->disc, (int64_t)Sc + s->B_r, GD);
  plan_partials(cv, pl, s, trunk, 1, GD);
  pl.rblocks = residual_blocks((int64_t)Sc * s->P);
  pl.rpart = cv.take((size_t)pl.rblocks * 8);
  pl.acc = cv.take((size_t)4 * 8 * GD);
  pl.hr = cv.take((size_t)Sc * s->P * 4);
  pl.hgn = cv.take((size_t)Sc * s->P * 4);
  pl.hdx = cv.take((size_t)Sc * pl.D.Kp * 4 * GD);
  if (s->lambda_gp > 0.0f) {
    pl.gpg = cv.take((size_t)Sc * s->disc.in_dim * 4 * GD);
    pl.gpp = cv.take((size_t)Sc * 8 * GD);
  }
  pl.total = round_up((int64_t)cv.off, 256);
}

// automatic chunking: the largest power-of-two share of the samples whose
// workspace fits in 128 GiB (under half of the 288 GB of HBM; larger chunks
// mean fewer, longer launches and fewer partial reductions)
static const size_t kAutoCap = (size_t)128 << 30;

static int choose_chunk(const pigan_step_desc* s, bool trunk = false, bool hier = false) {
  if (s->chunk_S > 0) return std::min(s->chunk_S, s->S);
  int Sc = s->S;
  StepPlan pl;
  while (true) {
    if (hier) plan_hier(s, Sc, pl, trunk);
    else plan_step(s, Sc, pl, trunk);
    if (pl.total <= kAutoCap || Sc == 1) return Sc;
    Sc = (Sc + 1) / 2;
  }
}

// gp_name: the entry point that takes the penalty's mixing weights
static pigan_status check_step(const pigan_step_desc* s, bool gp_entry = false,
                               const char* gp_name = "pigan_train_step_grads_gp") {
  if (!s) return fail(PIGAN_EINVAL, "null step descriptor");
  pigan_status st;
  if ((st = check_mlp(&s->genY, "genY")) != PIGAN_OK) return st;
  if ((st = check_mlp(&s->genU, "genU")) != PIGAN_OK) return st;
  if ((st = check_mlp(&s->disc, "disc")) != PIGAN_OK) return st;
  if ((st = check_dtype(s->dt)) != PIGAN_OK) return st;
  if (s->genU.n_groups != s->genY.n_groups || s->disc.n_groups != s->genY.n_groups)
    return fail(PIGAN_EINVAL, "n_groups differ between networks");
  if (s->d < 1 || s->d > 3) return fail(PIGAN_EINVAL, "d=%d must be 1, 2 or 3", s->d);
  if (s->n_z < 1) return fail(PIGAN_EINVAL, "n_z=%d must be >= 1", s->n_z);
  if (s->genY.in_dim != s->d + s->n_z || s->genU.in_dim != s->d + s->n_z)
    return fail(PIGAN_EINVAL, "generator in_dim must equal d + n_z = %d", s->d + s->n_z);
  if (s->S < 1 || s->P < 1) return fail(PIGAN_EINVAL, "S=%d and P=%d must be >= 1", s->S, s->P);
  if (s->n_sY < 1 || s->n_sU < 1) return fail(PIGAN_EINVAL, "n_sY=%d and n_sU=%d must be >= 1", s->n_sY, s->n_sU);
  if (s->disc.in_dim != s->n_sY + s->n_sU)
    return fail(PIGAN_EINVAL, "disc in_dim=%d must equal n_sY + n_sU = %d", s->disc.in_dim, s->n_sY + s->n_sU);
  if (s->B_r < 1) return fail(PIGAN_EINVAL, "B_r=%d must be >= 1", s->B_r);
  if (s->chunk_S < 0) return fail(PIGAN_EINVAL, "chunk_S=%d must be >= 0", s->chunk_S);
  if (!(s->lambda_pde >= 0.0f) || !__builtin_isfinite(s->lambda_pde))
    return fail(PIGAN_EINVAL, "lambda_pde must be finite and >= 0");
  if (!(s->lambda_gp >= 0.0f) || !__builtin_isfinite(s->lambda_gp))
    return fail(PIGAN_EINVAL, "lambda_gp must be finite and >= 0");
  if (!gp_entry && s->lambda_gp != 0.0f)
    return fail(PIGAN_ENOTSUP, "lambda_gp != 0 needs the per-pair mixing weights: use %s", gp_name);
  if (!(s->loss_scale > 0.0f) || !__builtin_isfinite(s->loss_scale))
    return fail(PIGAN_EINVAL, "loss_scale must be finite and > 0");
  if (s->critic_only != 0 && s->critic_only != 1)
    return fail(PIGAN_EINVAL, "critic_only=%d must be 0 or 1", s->critic_only);
  return PIGAN_OK;
}

// ---------------------------------------------------------------------------
// building blocks
// ---------------------------------------------------------------------------
template <class T> static T* tp(void* ws, size_t off) { return (T*)((char*)ws + off); }

template <class T>
static pigan_status gemm_nt(int epi, int nd1, int nd2, const NtArgs<T>& a, int G, hipStream_t st, const char* name) {
  const int C = 1 + nd1 + nd2;
  const double M = (double)C * a.seg.n_points;
  const int Ka = a.kx > 0 ? a.kx : a.K;   // the contraction the method defines (two-term weights: one term)
  const double flops = 2.0 * M * a.N * Ka * G + (a.y ? 2.0 * M * a.N * G : 0.0);
  const double es = sizeof(T);
  // operand X is read unless the first layer is formed in the kernel (then
  // its activations may be stored instead)
  double bytes = ((a.fp1 ? (a.f_out_h ? M * Ka : 0.0) : M * Ka) + (double)a.N * a.K) * es * G;
  if (epi == EPI_FWD) bytes += M * a.N * es * G * ((a.out_a ? 1 : 0) + (a.out_h ? 1 : 0)) + (a.y ? M * 4.0 * G : 0.0);
  else if (epi == EPI_BWD) bytes += (a.fp1 ? 1.0 : 2.0) * M * a.N * es * G;
  else bytes += M * a.N * 4.0 * G;
  // timing records are keyed by launch shape: one name = one kernel instantiation and size
  char key[64];
  snprintf(key, sizeof key, "%s_c%d_k%d_n%d%s%s", name, C, Ka, a.N, pm_tag(a.pm), a.kx > 0 ? "_w2" : "");
  ProfScope ps(st, key, flops, bytes);
  HIP_TRY(launch_gemm_nt<T>(epi, nd1, nd2, a, G, st));
  return PIGAN_OK;
}

// part: the plan's split-K partial buffer (fp32 entries, or fp64 for PM_SPLIT3)
template <class T>
static pigan_status weight_grad(const T* dA, int64_t a_g, int64_t lda, const T* H, int64_t h_g, int64_t ldh,
                                int64_t R, int64_t n_value, int N, int Jp, int J, float* gW, float* gb, int64_t g_g,
                                int accumulate, float scale, int32_t* nonfinite, void* part, double* pdb, int G,
                                hipStream_t st, int pm = PM_NATIVE) {
  int ns;
  int64_t rps;
  dw_split_plan(R, N, Jp, (int)sizeof(T), G, &ns, &rps);
  {
    char key[64];
    snprintf(key, sizeof key, "gemm_dw_n%d_j%d%s", N, Jp, pm_tag(pm));
    ProfScope ps(st, key, 2.0 * R * N * Jp * G,
                 ((double)R * (N + Jp) * sizeof(T) + (pm_wide(pm) ? 8.0 : 4.0) * ns * N * Jp) * G);
    HIP_TRY(launch_gemm_dw<T>(dA, a_g, lda, H, h_g, ldh, R, n_value, N, Jp, (float*)part, pdb, ns, rps, G, st, pm,
                              (double*)part));
  }
  {
    ProfScope ps(st, "reduce_dw", 0.0, (pm_wide(pm) ? 8.0 : 4.0) * ((double)ns + 1.0) * N * Jp * G);
    const int64_t nw = (int64_t)N * Jp;
    if (pm_wide(pm))
      HIP_TRY(launch_colsum<double>((double*)part, (int64_t)ns * nw, ns, nw, nw, Jp, J, gW, g_g, accumulate, scale,
                                    nonfinite, G, st));
    else
      HIP_TRY(launch_colsum<float>((float*)part, (int64_t)ns * nw, ns, nw, nw, Jp, J, gW, g_g, accumulate, scale,
                                   nonfinite, G, st));
    HIP_TRY(launch_colsum<double>(pdb, (int64_t)ns * N, ns, N, N, 1, 1, gb, g_g, accumulate, scale, nonfinite, G,
                                  st));
  }
  return PIGAN_OK;
}

// whether the collocation segment of a generator's chunk runs on the resident
// kernel (then the first and output layers are fused into the hidden GEMMs)
template <class T>
static bool colloc_resident(const NetBuf& nb) {
  const int W = nb.off.W;
  return nb.off.L >= 2 && !nb.skip && nb.heads == 1 &&
         nt_resident_ok((int)sizeof(T), nb.C(), W, W, nb.n_col, W, W);
}

// first-layer source of a second-layer GEMM (coordinates are per segment)
template <class T>
static void first_src(NtArgs<T>& a, const float* params, int64_t pg, int in_dim, int d, const float* zp,
                      int64_t zp_g) {
  a.fp1 = params; a.fp_g = pg; a.f_in = in_dim; a.f_d = d;
  a.fzp = zp; a.fzp_g = zp_g;
}

// collocation forward weights of hidden layer l: two-term rows [W_hi | W_lo]
// in 16-bit storage
template <class T>
static void colloc_weights(NtArgs<T>& a, void* ws, const NetBuf& nb, int l) {
  const int W = nb.off.W, L = nb.off.L;
  const int tw = two_term<T>() ? 2 : 1;
  a.Wm = tp<T>(ws, nb.wc) + (size_t)(l - 2) * W * W * tw;
  a.w_g = (int64_t)std::max(L - 1, 1) * W * W * tw;
  a.ldw = (int64_t)W * tw;
  a.K = W * tw;
  a.kx = tw == 2 ? W : 0;
}

// Forward of one generator over a chunk: sensor rows, then (unless colloc is
// false: a critic-only step of the paired or trunk generators) collocation rows.
template <class T>
static pigan_status gen_chunk_fwd(void* ws, const NetBuf& nb, const float* params, const float* xs, int64_t xs_g,
                                  const float* xc, int64_t xc_g, const float* z, int64_t z_g, int d, int n_z, int Sc,
                                  int P, int G, hipStream_t st, bool colloc = true) {
  const int W = nb.off.W, L = nb.off.L;
  const int64_t pg = nb.off.n;
  const int64_t ags = nb.Rs * W, agc = nb.Rc * W;   // per-group element strides of the activations
  {
    ProfScope ps(st, "zproj", 2.0 * Sc * W * n_z * G, 0.0);
    HIP_TRY(launch_zproj(params, pg, nb.off.in_dim, d, W, z, z_g, n_z, Sc, tp<float>(ws, nb.zp), (int64_t)Sc * W, G,
                         st));
  }
  // ---- sensor rows: fp32 storage, split products, value stream only
  {
    FirstArgs<float> fa{};
    fa.p1 = params; fa.p_g = pg; fa.in_dim = nb.off.in_dim; fa.d = d; fa.W = W;
    fa.zp = tp<float>(ws, nb.zp); fa.zp_g = (int64_t)Sc * W;
    fa.out_a = tp<float>(ws, nb.As[1]); fa.out_h = tp<float>(ws, nb.Hs[1]); fa.o_g = ags; fa.ldo = W;
    fa.x = xs; fa.x_g = xs_g; fa.x_shared = 1; fa.Pn = nb.n_s;
    fa.seg = Seg{nb.n_sen, 0, 0};
    fa.exact = adv_pm<T>() == PM_F64;
    ProfScope ps(st, "first_fwd", 2.0 * nb.n_sen * W * d * G, (double)nb.n_sen * W * 2 * 4 * G);
    HIP_TRY(launch_first_fwd<float>(0, 0, fa, G, st));
  }
  for (int l = 2; l <= L; ++l) {
    NtArgs<float> a{};
    a.X = tp<float>(ws, nb.Hs[l - 1]); a.x_g = ags; a.ldx = W;
    a.Wm = tp<float>(ws, nb.ws) + (size_t)(l - 2) * W * W; a.w_g = (int64_t)std::max(L - 1, 1) * W * W; a.ldw = W;
    a.bias = params + nb.off.b[l]; a.b_g = pg;
    a.out_a = tp<float>(ws, nb.As[l]); a.out_h = tp<float>(ws, nb.Hs[l]); a.o_g = ags; a.ldo = W;
    if (nb.skip && trunk_skip(l)) a.skip = tp<float>(ws, nb.Hs[l - 2]);   // residual block output
    a.N = W; a.K = W; a.pm = adv_pm<T>();
    a.seg = Seg{nb.n_sen, 0, 0};
    pigan_status s1 = gemm_nt<float>(EPI_FWD, 0, 0, a, G, st, "gemm_fwd");
    if (s1 != PIGAN_OK) return s1;
  }
  {
    ProfScope ps(st, "out_fwd", 2.0 * nb.heads * nb.n_sen * W * G, (double)nb.heads * nb.n_sen * W * 4 * G);
    HIP_TRY(launch_out_fwd<float>(tp<float>(ws, nb.Hs[L]), ags, W, nb.n_sen, nb.n_sen, W, params + nb.off.wout, pg,
                                  tp<float>(ws, nb.jet), nb.R, G, st));
    if (nb.heads == 2)   // second head (u): [w_u, b_u] follows [w_Y, b_Y]
      HIP_TRY(launch_out_fwd<float>(tp<float>(ws, nb.Hs[L]), ags, W, nb.n_sen, nb.n_sen, W,
                                    params + nb.off.wout + W + 1, pg, tp<float>(ws, nb.jet2), nb.R, G, st));
  }
  if (!colloc) return PIGAN_OK;
  // ---- collocation rows: storage type T, every jet stream
  const int C = nb.C();
  const int64_t mc = C * nb.n_col;
  const bool resident = colloc_resident<T>(nb);
  if (!resident) {
    FirstArgs<T> fa{};
    fa.p1 = params; fa.p_g = pg; fa.in_dim = nb.off.in_dim; fa.d = d; fa.W = W;
    fa.zp = tp<float>(ws, nb.zp); fa.zp_g = (int64_t)Sc * W;
    fa.out_a = tp<T>(ws, nb.Ac[1]); fa.out_h = tp<T>(ws, nb.Hc[1]); fa.o_g = agc; fa.ldo = W;
    fa.x = xc; fa.x_g = xc_g; fa.x_shared = 0; fa.Pn = P;
    fa.seg = Seg{nb.n_col, 0, nb.n_col};
    fa.exact = sizeof(T) == 4;
    ProfScope ps(st, "first_fwd", 2.0 * nb.n_col * W * d * G, (double)mc * W * 2 * sizeof(T) * G);
    HIP_TRY(launch_first_fwd<T>(nb.nd1, nb.nd2, fa, G, st));
  }
  for (int l = 2; l <= L; ++l) {
    NtArgs<T> a{};
    a.X = tp<T>(ws, nb.Hc[l - 1]); a.x_g = agc; a.ldx = W;
    colloc_weights<T>(a, ws, nb, l);
    a.bias = params + nb.off.b[l]; a.b_g = pg;
    a.out_a = tp<T>(ws, nb.Ac[l]); a.out_h = tp<T>(ws, nb.Hc[l]); a.o_g = agc; a.ldo = W;
    if (l == L && resident) {
      a.out_h = nullptr;
      a.y = tp<float>(ws, nb.jet) + nb.n_sen; a.y_g = nb.R; a.wout = params + nb.off.wout; a.wo_g = pg;
    }
    if (l == 2 && resident) {
      first_src(a, params, pg, nb.off.in_dim, d, tp<float>(ws, nb.zp), (int64_t)Sc * W);
      a.f_out_h = tp<T>(ws, nb.Hc[1]);
    }
    if (nb.skip && trunk_skip(l)) a.skip = tp<T>(ws, nb.Hc[l - 2]);
    a.N = W;
    a.seg = Seg{nb.n_col, 0, nb.n_col};
    a.fx = xc; a.fx_g = xc_g; a.fx_shared = 0; a.fPn = P;
    pigan_status s1 = gemm_nt<T>(EPI_FWD, nb.nd1, nb.nd2, a, G, st, "gemm_fwd");
    if (s1 != PIGAN_OK) return s1;
  }
  if (!resident) {
    ProfScope ps(st, "out_fwd", 2.0 * nb.heads * mc * W * G, (double)nb.heads * mc * W * sizeof(T) * G);
    HIP_TRY(launch_out_fwd<T>(tp<T>(ws, nb.Hc[L]), agc, W, mc, nb.n_col, W, params + nb.off.wout, pg,
                              tp<float>(ws, nb.jet) + nb.n_sen, nb.R, G, st));
    if (nb.heads == 2)
      HIP_TRY(launch_out_fwd<T>(tp<T>(ws, nb.Hc[L]), agc, W, mc, nb.n_col, W, params + nb.off.wout + W + 1, pg,
                                tp<float>(ws, nb.jet2) + nb.n_sen, nb.R, G, st));
  }
  return PIGAN_OK;
}

// Reverse pass of one generator over a chunk (cotangents of the outputs are
// in nb.gbar).  Gradients go to grad (accumulated when accumulate != 0).
template <class T>
static pigan_status gen_chunk_bwd(void* ws, const StepPlan& pl, const NetBuf& nb, const float* params,
                                  const float* xs, int64_t xs_g, const float* xc, int64_t xc_g, const float* z,
                                  int64_t z_g, int d, int n_z, int Sc, int P, float* grad, int accumulate, float scale,
                                  int32_t* nonfinite, int G, hipStream_t st) {
  const int W = nb.off.W, L = nb.off.L;
  const int64_t pg = nb.off.n;
  const int64_t ags = nb.Rs * W, agc = nb.Rc * W;
  const int C = nb.C();
  const int64_t mc = C * nb.n_col;
  const int pm = adv_pm<T>();
  const bool resident = colloc_resident<T>(nb);
  const int blk_sen = out_bwd_blocks(nb.n_sen, (int)nb.ppb_sen);
  const int n_slots = blk_sen + out_bwd_blocks(nb.n_col, (int)nb.ppb_col);
  // output layer of both segments: one slot range of w_out partials
  if (nb.heads == 2) {
    // two heads on the trunk's last activations; their cotangent is also the
    // skip cotangent of the top residual block's input
    const bool topskip = nb.skip && trunk_skip(L);
    Out2BwdArgs<float> os{};
    os.A = tp<float>(ws, nb.As[L]); os.H = tp<float>(ws, nb.Hs[L]); os.dA = tp<float>(ws, nb.dAs[0]);
    os.gh = topskip ? tp<float>(ws, nb.ghs) : nullptr;
    os.o_g = ags; os.ldo = W;
    os.gbar0 = tp<float>(ws, nb.gbar); os.gbar1 = tp<float>(ws, nb.gbar2); os.gb_g = nb.R;
    os.wout = params + nb.off.wout; os.w_g = pg;
    os.W = W; os.part = tp<double>(ws, nb.ob); os.n_slots = n_slots;
    os.ppb = nb.ppb_sen; os.slot0 = 0; os.seg = Seg{nb.n_sen, 0, 0}; os.exact = pm == PM_F64;
    Out2BwdArgs<T> oc{};
    oc.A = tp<T>(ws, nb.Ac[L]); oc.H = tp<T>(ws, nb.Hc[L]); oc.dA = tp<T>(ws, nb.dAc[0]);
    oc.gh = topskip ? tp<T>(ws, nb.ghc) : nullptr;
    oc.o_g = agc; oc.ldo = W;
    oc.gbar0 = tp<float>(ws, nb.gbar) + nb.n_sen; oc.gbar1 = tp<float>(ws, nb.gbar2) + nb.n_sen; oc.gb_g = nb.R;
    oc.wout = params + nb.off.wout; oc.w_g = pg;
    oc.W = W; oc.part = tp<double>(ws, nb.ob); oc.n_slots = n_slots;
    oc.ppb = nb.ppb_col; oc.slot0 = blk_sen; oc.seg = Seg{nb.n_col, 0, nb.n_col}; oc.exact = sizeof(T) == 4;
    ProfScope ps(st, "out_bwd", 0.0,
                 ((double)nb.n_sen * 4 + (double)mc * sizeof(T)) * W * (topskip ? 4 : 3) * G);
    HIP_TRY(launch_out2_bwd<float>(0, 0, os, G, st));
    HIP_TRY(launch_out2_bwd<T>(nb.nd1, nb.nd2, oc, G, st));
    HIP_TRY(launch_colsum<double>(tp<double>(ws, nb.ob), (int64_t)n_slots * 2 * (W + 1), n_slots, 2 * (W + 1),
                                  2 * (W + 1), 1, 1, grad + nb.off.wout, pg, accumulate, scale, nonfinite, G, st));
  } else {
    OutBwdArgs<float> os{};
    os.A = tp<float>(ws, nb.As[L]); os.dA = tp<float>(ws, nb.dAs[0]); os.o_g = ags; os.ldo = W;
    os.gbar = tp<float>(ws, nb.gbar); os.gb_g = nb.R;
    os.wout = params + nb.off.wout; os.w_g = pg;
    os.W = W; os.part = tp<double>(ws, nb.ob); os.n_slots = n_slots;
    os.ppb = nb.ppb_sen; os.slot0 = 0; os.seg = Seg{nb.n_sen, 0, 0}; os.exact = pm == PM_F64;
    OutBwdArgs<T> oc{};
    oc.A = tp<T>(ws, nb.Ac[L]); oc.dA = tp<T>(ws, nb.dAc[0]); oc.o_g = agc; oc.ldo = W;
    oc.gbar = tp<float>(ws, nb.gbar) + nb.n_sen; oc.gb_g = nb.R;
    oc.wout = params + nb.off.wout; oc.w_g = pg;
    oc.W = W; oc.part = tp<double>(ws, nb.ob); oc.n_slots = n_slots;
    oc.ppb = nb.ppb_col; oc.slot0 = blk_sen; oc.seg = Seg{nb.n_col, 0, nb.n_col}; oc.exact = sizeof(T) == 4;
    ProfScope ps(st, "out_bwd", 0.0, ((double)nb.n_sen * 4 + (double)mc * sizeof(T)) * W * 2 * G);
    HIP_TRY(launch_out_bwd<float>(0, 0, os, G, st));
    HIP_TRY(launch_out_bwd<T>(nb.nd1, nb.nd2, oc, G, st));
    HIP_TRY(launch_colsum<double>(tp<double>(ws, nb.ob), (int64_t)n_slots * (W + 1), n_slots, W + 1, W + 1, 1, 1,
                                  grad + nb.off.wout, pg, accumulate, scale, nonfinite, G, st));
  }
  void* part = tp<void>(ws, pl.dwp);
  double* pdb = tp<double>(ws, pl.dwdb);
  int cur = 0;
  for (int l = L; l >= 2; --l) {
    // weight and bias gradients: sensor rows (split products), then the
    // collocation rows added
    pigan_status s1 = weight_grad<float>(tp<float>(ws, nb.dAs[cur]), ags, W, tp<float>(ws, nb.Hs[l - 1]), ags, W,
                                         nb.n_sen, nb.n_sen, W, W, W, grad + nb.off.w[l], grad + nb.off.b[l], pg,
                                         accumulate, scale, nonfinite, part, pdb, G, st, pm);
    if (s1 != PIGAN_OK) return s1;
    s1 = weight_grad<T>(tp<T>(ws, nb.dAc[cur]), agc, W, tp<T>(ws, nb.Hc[l - 1]), agc, W, mc, nb.n_col, W, W, W,
                        grad + nb.off.w[l], grad + nb.off.b[l], pg, 1, scale, nonfinite, part, pdb, G, st);
    if (s1 != PIGAN_OK) return s1;
    // h_{l-1} is a residual block's input (when l + 1 <= L): add the total
    // cotangent of that block's output; when h_{l-1} is itself a block's
    // output (l - 1 >= 3), keep its total for the block below (in place)
    const bool skip_in = nb.skip && (l - 1) % 2 == 1 && l + 1 <= L;
    const bool skip_out = nb.skip && (l - 1) % 2 == 1 && l - 1 >= 3;
    NtArgs<float> as{};
    as.X = tp<float>(ws, nb.dAs[cur]); as.x_g = ags; as.ldx = W;
    as.Wm = tp<float>(ws, nb.wsT) + (size_t)(l - 2) * W * W; as.w_g = (int64_t)std::max(L - 1, 1) * W * W; as.ldw = W;
    as.aprev = tp<float>(ws, nb.As[l - 1]); as.out_da = tp<float>(ws, nb.dAs[1 - cur]); as.o_g = ags; as.ldo = W;
    if (skip_in) as.skip_g = tp<float>(ws, nb.ghs);
    if (skip_out) as.out_gh = tp<float>(ws, nb.ghs);
    as.N = W; as.K = W; as.pm = pm;
    as.seg = Seg{nb.n_sen, 0, 0};
    if ((s1 = gemm_nt<float>(EPI_BWD, 0, 0, as, G, st, "gemm_bwd")) != PIGAN_OK) return s1;
    NtArgs<T> ac{};
    ac.X = tp<T>(ws, nb.dAc[cur]); ac.x_g = agc; ac.ldx = W;
    ac.Wm = tp<T>(ws, nb.wcT) + (size_t)(l - 2) * W * W; ac.w_g = (int64_t)std::max(L - 1, 1) * W * W; ac.ldw = W;
    ac.aprev = tp<T>(ws, nb.Ac[l - 1]); ac.out_da = tp<T>(ws, nb.dAc[1 - cur]); ac.o_g = agc; ac.ldo = W;
    if (l == 2 && resident)   // the first layer's pre-activations were never stored
      first_src(ac, params, pg, nb.off.in_dim, d, tp<float>(ws, nb.zp), (int64_t)Sc * W);
    if (skip_in) ac.skip_g = tp<T>(ws, nb.ghc);
    if (skip_out) ac.out_gh = tp<T>(ws, nb.ghc);
    ac.N = W; ac.K = W;
    ac.seg = Seg{nb.n_col, 0, nb.n_col};
    ac.fx = xc; ac.fx_g = xc_g; ac.fx_shared = 0; ac.fPn = P;
    if ((s1 = gemm_nt<T>(EPI_BWD, nb.nd1, nb.nd2, ac, G, st, "gemm_bwd")) != PIGAN_OK) return s1;
    cur = 1 - cur;
  }
  FirstBwdArgs<T> fb{};
  fb.dAs = tp<float>(ws, nb.dAs[cur]); fb.as_g = ags; fb.ldas = W;
  fb.dA = tp<T>(ws, nb.dAc[cur]); fb.a_g = agc; fb.lda = W;
  fb.n_sen = nb.n_sen; fb.n_col = nb.n_col; fb.n_s = nb.n_s; fb.P = P; fb.S = Sc; fb.W = W; fb.d = d; fb.nd1 = nb.nd1;
  fb.xs = xs; fb.xs_g = xs_g; fb.xc = xc; fb.xc_g = xc_g; fb.part = tp<double>(ws, nb.fb);
  fb.nrc = nb.nrc;   // planned for the largest chunk: Sc * nrc never exceeds the partial buffer
  {
    ProfScope ps(st, "first_bwd", 0.0, ((double)nb.n_sen * 4 + (double)(1 + nb.nd1) * nb.n_col * sizeof(T)) * W * G);
    HIP_TRY(launch_first_bwd<T>(fb, G, st));
    HIP_TRY(launch_first_wgrad(tp<double>(ws, nb.fb), Sc, fb.nrc, W, d, nb.nd1, nb.off.in_dim, z, z_g, n_z, grad, pg,
                               accumulate, scale, nonfinite, G, st));
  }
  return PIGAN_OK;
}

template <class T>
static pigan_status cast_gen_weights(void* ws, const NetBuf& nb, const float* params, int G, hipStream_t st) {
  const int W = nb.off.W, L = nb.off.L;
  const int64_t dg = (int64_t)std::max(L - 1, 1) * W * W;
  for (int l = 2; l <= L; ++l) {
    const float* src = params + nb.off.w[l];
    const size_t o = (size_t)(l - 2) * W * W;
    if constexpr (two_term<T>()) {
      HIP_TRY(launch_cast2<T>(src, nb.off.n, W, W, tp<T>(ws, nb.wc) + 2 * o, 2 * dg, G, st));
      HIP_TRY(launch_cast<T>(src, nb.off.n, W, W, W, nullptr, tp<T>(ws, nb.wcT) + o, dg, G, st));
    } else {
      HIP_TRY(launch_cast<T>(src, nb.off.n, W, W, W, tp<T>(ws, nb.wc) + o, tp<T>(ws, nb.wcT) + o, dg, G, st));
    }
    // the sensor rows' copies: pre-split for the split products
    if constexpr (adv_pm<T>() == PM_SPLIT2)
      HIP_TRY(launch_cast_pair(src, nb.off.n, W, W, W, tp<float>(ws, nb.ws) + o, tp<float>(ws, nb.wsT) + o, dg, G,
                               st));
    else
      HIP_TRY(launch_cast<float>(src, nb.off.n, W, W, W, tp<float>(ws, nb.ws) + o, tp<float>(ws, nb.wsT) + o, dg, G,
                                 st));
  }
  return PIGAN_OK;
}

// the critic's padded first-layer weights and their transpose, and the
// hidden layers' weights and transposes (fp32 copies with aligned rows;
// pair: pre-split for the split products)
static pigan_status cast_disc_weights(void* ws, const DiscBuf& D, const float* pD, int WD, int LD, int n_in, int G,
                                      hipStream_t st, bool pair) {
  auto cast = [&](const float* src, int N, int K, int Kp, float* dst, float* dstT, int64_t d_g) {
    return pair ? launch_cast_pair(src, D.off.n, N, K, Kp, dst, dstT, d_g, G, st)
                : launch_cast<float>(src, D.off.n, N, K, Kp, dst, dstT, d_g, G, st);
  };
  HIP_TRY(cast(pD + D.off.w[1], WD, n_in, D.Kp, tp<float>(ws, D.w1), tp<float>(ws, D.w1T), (int64_t)WD * D.Kp));
  const int64_t dgl = (int64_t)std::max(LD - 1, 1) * WD * WD;
  for (int l = 2; l <= LD; ++l)
    HIP_TRY(cast(pD + D.off.w[l], WD, WD, WD, tp<float>(ws, D.wc) + (size_t)(l - 2) * WD * WD,
                 tp<float>(ws, D.wcT) + (size_t)(l - 2) * WD * WD, dgl));
  return PIGAN_OK;
}

// critic forward over `seg` (nd1 = 1: value and one tangent stream)
static pigan_status disc_forward(void* ws, const DiscBuf& D, const float* pD, int WD, int LD, Seg seg, int nd1,
                                 int G, hipStream_t st, const char* name, int pm) {
  const int64_t dact = D.Bmax * WD;
  for (int l = 1; l <= LD; ++l) {
    NtArgs<float> a{};
    if (l == 1) {
      a.X = tp<float>(ws, D.X0); a.x_g = D.Bmax * D.Kp; a.ldx = D.Kp;
      a.Wm = tp<float>(ws, D.w1); a.w_g = (int64_t)WD * D.Kp; a.ldw = D.Kp; a.K = D.Kp;
    } else {
      a.X = tp<float>(ws, D.H[l - 1]); a.x_g = dact; a.ldx = WD;
      a.Wm = tp<float>(ws, D.wc) + (size_t)(l - 2) * WD * WD; a.w_g = (int64_t)std::max(LD - 1, 1) * WD * WD;
      a.ldw = WD; a.K = WD;
    }
    a.bias = pD + D.off.b[l]; a.b_g = D.off.n;
    a.out_a = tp<float>(ws, D.A[l]); a.out_h = tp<float>(ws, D.H[l]); a.o_g = dact; a.ldo = WD;
    a.N = WD; a.pm = pm;
    a.seg = seg;
    pigan_status r = gemm_nt<float>(EPI_FWD, nd1, 0, a, G, st, name);
    if (r != PIGAN_OK) return r;
  }
  return PIGAN_OK;
}

// Critic gradient penalty on n pairs of this chunk, whose interpolates
// x_b = eps_b R_b + (1 - eps_b) F_b the caller has written to the critic's
// input rows [0, n):  P = w lambda_gp / n_gp sum_b (|g_b| - 1)^2 with
// g_b = dD/dv at x_b.  dP/dphi = sum_b c_b . dg_b/dphi with c_b = dP/dg_b
// fixed, and c_b . g_b is the directional derivative of D at x_b along c_b:
// so the weight gradient is the reverse pass of a (value, tangent) jet of D
// seeded with (x_b, c_b), with cotangent 1 on the tangent output.  Added to
// gD; the row terms go to acc[g][3].  G critics, one per grid z.
static pigan_status critic_penalty(void* ws, const StepPlan& pl, const pigan_step_desc* s, const float* pD,
                                   const float* w_group, int n, float* gD, float inv, int32_t* nonfinite,
                                   double* acc, int G, hipStream_t st, int pm) {
  const DiscBuf& D = pl.D;
  const int WD = s->disc.width, LD = s->disc.n_hidden, n_in = s->disc.in_dim;
  const int64_t dact = D.Bmax * WD, xg = D.Bmax * D.Kp;
  const int n_gp = std::min(s->S, s->B_r);
  const int64_t gg = (int64_t)pl.Sc * n_in;
  void* part = tp<void>(ws, pl.dwp);
  double* pdb = tp<double>(ws, pl.dwdb);
  pigan_status r;
  {
    ProfScope ps(st, "gp_misc", 0.0, 0.0);
    HIP_TRY(launch_fill2(tp<float>(ws, D.seed), D.Bmax, n, 1.0f, 0.0f, 0, G, st));
  }
  // 1. D on the interpolates, then its reverse pass to the input: g = dD/dv
  if ((r = disc_forward(ws, D, pD, WD, LD, Seg{n, 0, 0}, 0, G, st, "gp_fwd", pm)) != PIGAN_OK) return r;
  OutBwdArgs<float> ob{};
  ob.A = tp<float>(ws, D.A[LD]); ob.dA = tp<float>(ws, D.dA[0]); ob.o_g = dact; ob.ldo = WD;
  ob.gbar = tp<float>(ws, D.seed); ob.gb_g = D.Bmax;
  ob.wout = pD + D.off.wout; ob.w_g = D.off.n;
  ob.W = WD; ob.ppb = D.ppb; ob.part = tp<double>(ws, D.ob); ob.n_slots = out_bwd_blocks(n, (int)D.ppb);
  ob.slot0 = 0; ob.seg = Seg{n, 0, 0}; ob.exact = pm == PM_F64;
  {
    ProfScope ps(st, "gp_bwd", 0.0, (double)n * WD * 2 * 4 * G);
    HIP_TRY(launch_out_bwd<float>(0, 0, ob, G, st));   // (its output-weight partials are not used)
  }
  int cur = 0;
  for (int l = LD; l >= 2; --l) {
    NtArgs<float> a{};
    a.X = tp<float>(ws, D.dA[cur]); a.x_g = dact; a.ldx = WD;
    a.Wm = tp<float>(ws, D.wcT) + (size_t)(l - 2) * WD * WD; a.w_g = (int64_t)std::max(LD - 1, 1) * WD * WD;
    a.ldw = WD;
    a.aprev = tp<float>(ws, D.A[l - 1]); a.out_da = tp<float>(ws, D.dA[1 - cur]); a.o_g = dact; a.ldo = WD;
    a.N = WD; a.K = WD; a.pm = pm; a.seg = Seg{n, 0, 0};
    if ((r = gemm_nt<float>(EPI_BWD, 0, 0, a, G, st, "gp_bwd")) != PIGAN_OK) return r;
    cur = 1 - cur;
  }
  {
    NtArgs<float> a{};
    a.X = tp<float>(ws, D.dA[cur]); a.x_g = dact; a.ldx = WD;
    a.Wm = tp<float>(ws, D.w1T); a.w_g = (int64_t)WD * D.Kp; a.ldw = WD;
    a.N = D.Kp; a.K = WD; a.pm = pm; a.seg = Seg{n, 0, 0};
    a.seedY = tp<float>(ws, pl.gpg); a.sY_g = gg; a.seedU = nullptr; a.sU_g = 0;
    a.nY = n_in; a.nU = 0; a.df_sign = 1.0f;
    if ((r = gemm_nt<float>(EPI_DF, 0, 0, a, G, st, "gp_bwd")) != PIGAN_OK) return r;
  }
  // 2. row terms (|g| - 1)^2 and tangent rows c = dP/dg (times the loss scale)
  {
    ProfScope ps(st, "gp_misc", 0.0, 0.0);
    const float scale = (float)(2.0 * s->lambda_gp * s->loss_scale / n_gp);
    HIP_TRY(launch_gp_norm<float>(tp<float>(ws, pl.gpg), gg, n, n_in, w_group, scale, tp<double>(ws, pl.gpp), n,
                                  tp<float>(ws, D.X0), xg, D.Kp, G, st));
    HIP_TRY(launch_sum_partials(tp<double>(ws, pl.gpp), n, acc, 4, 3, G, st));
    HIP_TRY(launch_fill2(tp<float>(ws, D.seed), D.Bmax, n, 0.0f, 1.0f, 1, G, st));
  }
  // 3. (value, tangent) jet of D and its reverse pass with cotangent 1 on the
  //    tangent output: the weight gradient of the penalty
  if ((r = disc_forward(ws, D, pD, WD, LD, Seg{n, 0, n}, 1, G, st, "gp_fwd", pm)) != PIGAN_OK) return r;
  ob.A = tp<float>(ws, D.A[LD]); ob.dA = tp<float>(ws, D.dA[0]);
  ob.n_slots = out_bwd_blocks(n, (int)D.ppb);     // blocks run over points, every stream of a point in one
  ob.seg = Seg{n, 0, n};
  {
    ProfScope ps(st, "gp_bwd", 0.0, (double)2 * n * WD * 2 * 4 * G);
    HIP_TRY(launch_out_bwd<float>(1, 0, ob, G, st));
    HIP_TRY(launch_colsum<double>(tp<double>(ws, D.ob), (int64_t)ob.n_slots * (WD + 1), ob.n_slots, WD + 1, WD + 1,
                                  1, 1, gD + D.off.wout, D.off.n, 1, inv, nonfinite, G, st));
  }
  cur = 0;
  for (int l = LD; l >= 2; --l) {
    if ((r = weight_grad<float>(tp<float>(ws, D.dA[cur]), dact, WD, tp<float>(ws, D.H[l - 1]), dact, WD,
                                2 * (int64_t)n, n, WD, WD, WD, gD + D.off.w[l], gD + D.off.b[l], D.off.n, 1, inv,
                                nonfinite, part, pdb, G, st, pm)) != PIGAN_OK)
      return r;
    NtArgs<float> a{};
    a.X = tp<float>(ws, D.dA[cur]); a.x_g = dact; a.ldx = WD;
    a.Wm = tp<float>(ws, D.wcT) + (size_t)(l - 2) * WD * WD; a.w_g = (int64_t)std::max(LD - 1, 1) * WD * WD;
    a.ldw = WD;
    a.aprev = tp<float>(ws, D.A[l - 1]); a.out_da = tp<float>(ws, D.dA[1 - cur]); a.o_g = dact; a.ldo = WD;
    a.N = WD; a.K = WD; a.pm = pm; a.seg = Seg{n, 0, n};
    if ((r = gemm_nt<float>(EPI_BWD, 1, 0, a, G, st, "gp_bwd")) != PIGAN_OK) return r;
    cur = 1 - cur;
  }
  return weight_grad<float>(tp<float>(ws, D.dA[cur]), dact, WD, tp<float>(ws, D.X0), xg, D.Kp, 2 * (int64_t)n, n, WD,
                            D.Kp, n_in, gD + D.off.w[1], gD + D.off.b[1], D.off.n, 1, inv, nonfinite, part, pdb, G,
                            st, pm);
}

// Critic forward on the B rows of D.X0 (fake rows first, then n_real real
// rows), its seeds (+w/S fake, -w/B_r real, times the loss scale) and the
// reverse pass with every weight gradient (accumulated when accum != 0).  On
// return D.dA[*cur] holds the first layer's pre-activation cotangents.
static pigan_status disc_pass(void* ws, const StepPlan& pl, const float* pD, int WD, int LD, int n_in, int B, int Sc,
                              int n_real, int S, int B_r, const float* w_group, float ls, float inv, int accum,
                              float* gD, int32_t* nonfinite, double* acc, int G, hipStream_t st, int* cur_out,
                              int pm) {
  const DiscBuf& D = pl.D;
  const int64_t dact = D.Bmax * WD;
  void* part = tp<void>(ws, pl.dwp);
  double* pdb = tp<double>(ws, pl.dwdb);
  pigan_status r;
  if ((r = disc_forward(ws, D, pD, WD, LD, Seg{B, 0, 0}, 0, G, st, "disc_fwd", pm)) != PIGAN_OK) return r;
  {
    ProfScope ps(st, "out_fwd", 2.0 * B * WD * G, (double)B * WD * 4 * G);
    HIP_TRY(launch_out_fwd<float>(tp<float>(ws, D.H[LD]), dact, WD, B, B, WD, pD + D.off.wout, D.off.n,
                                  tp<float>(ws, D.score), D.Bmax, G, st));
    HIP_TRY(launch_disc_seed(tp<float>(ws, D.score), D.Bmax, Sc, n_real, S, B_r, w_group, ls,
                             tp<float>(ws, D.seed), acc, 4, G, st));
  }
  // critic reverse pass
  {
    OutBwdArgs<float> ob{};
    ob.A = tp<float>(ws, D.A[LD]); ob.dA = tp<float>(ws, D.dA[0]); ob.o_g = dact; ob.ldo = WD;
    ob.gbar = tp<float>(ws, D.seed); ob.gb_g = D.Bmax;
    ob.wout = pD + D.off.wout; ob.w_g = D.off.n;
    ob.W = WD; ob.ppb = D.ppb; ob.part = tp<double>(ws, D.ob); ob.n_slots = out_bwd_blocks(B, (int)D.ppb);
    ob.slot0 = 0; ob.seg = Seg{B, 0, 0}; ob.exact = pm == PM_F64;
    ProfScope ps(st, "out_bwd", 0.0, (double)B * WD * 2 * 4 * G);
    HIP_TRY(launch_out_bwd<float>(0, 0, ob, G, st));
    HIP_TRY(launch_colsum<double>(tp<double>(ws, D.ob), (int64_t)ob.n_slots * (WD + 1), ob.n_slots, WD + 1, WD + 1,
                                  1, 1, gD + D.off.wout, D.off.n, accum, inv, nonfinite, G, st));
  }
  int cur = 0;
  for (int l = LD; l >= 2; --l) {
    if ((r = weight_grad<float>(tp<float>(ws, D.dA[cur]), dact, WD, tp<float>(ws, D.H[l - 1]), dact, WD, B, B, WD, WD,
                                WD, gD + D.off.w[l], gD + D.off.b[l], D.off.n, accum, inv, nonfinite, part, pdb, G, st,
                                pm)) != PIGAN_OK)
      return r;
    NtArgs<float> a{};
    a.X = tp<float>(ws, D.dA[cur]); a.x_g = dact; a.ldx = WD;
    a.Wm = tp<float>(ws, D.wcT) + (size_t)(l - 2) * WD * WD; a.w_g = (int64_t)std::max(LD - 1, 1) * WD * WD;
    a.ldw = WD;
    a.aprev = tp<float>(ws, D.A[l - 1]); a.out_da = tp<float>(ws, D.dA[1 - cur]); a.o_g = dact; a.ldo = WD;
    a.N = WD; a.K = WD; a.pm = pm; a.seg = Seg{B, 0, 0};
    if ((r = gemm_nt<float>(EPI_BWD, 0, 0, a, G, st, "disc_bwd")) != PIGAN_OK) return r;
    cur = 1 - cur;
  }
  if ((r = weight_grad<float>(tp<float>(ws, D.dA[cur]), dact, WD, tp<float>(ws, D.X0), D.Bmax * D.Kp, D.Kp, B, B, WD,
                              D.Kp, n_in, gD + D.off.w[1], gD + D.off.b[1], D.off.n, accum, inv, nonfinite, part, pdb,
                              G, st, pm)) != PIGAN_OK)
    return r;
  *cur_out = cur;
  return PIGAN_OK;
}

// chunk-local view of a network's buffers: the plan is laid out for pl.Sc
// samples; a shorter last chunk uses the same buffers with its own row counts
static NetBuf chunk_view(const NetBuf& nb, int Sc, int P) {
  NetBuf c = nb;
  c.n_sen = (int64_t)Sc * c.n_s;
  c.n_col = (int64_t)Sc * P;
  c.rows = c.n_sen + c.C() * c.n_col;
  return c;
}

template <class T>
static pigan_status run_step(const pigan_step_desc* s, const StepPlan& pl, const float* pY, const float* pU,
                             const float* pD, const float* z, const float* xc, const float* xsY, const float* xsU,
                             const float* f, float f_const, const float* real, const float* w_group, float* gY,
                             float* gU, float* gD, float* loss, int32_t* nonfinite, void* ws, hipStream_t st,
                             const float* gp_eps, float* gp) {
  const int G = pl.G, d = s->d, n_z = s->n_z, P = s->P, S = s->S;
  const float ls = s->loss_scale;
  const float inv = 1.0f / ls;
  const DiscBuf& D = pl.D;
  const int WD = s->disc.width, LD = s->disc.n_hidden, n_in = s->disc.in_dim;
  const int pm = adv_pm<T>();
  double* acc = tp<double>(ws, pl.acc);
  pigan_status r;

  {
    ProfScope ps(st, "misc", 0.0, 0.0);
    HIP_TRY(launch_zero(acc, 4 * G, nonfinite, st));
    if ((r = cast_gen_weights<T>(ws, pl.Y, pY, G, st)) != PIGAN_OK) return r;
    if (!pl.trunk && (r = cast_gen_weights<T>(ws, pl.U, pU, G, st)) != PIGAN_OK) return r;
    if (pl.trunk)   // the trunk sees both sensor sets: locations [Y sensors ; u sensors]
      HIP_TRY(launch_concat_rows(xsY, (int64_t)s->n_sY * d, s->n_sY, xsU, (int64_t)s->n_sU * d, s->n_sU, d,
                                 tp<float>(ws, pl.Y.xsc), (int64_t)(s->n_sY + s->n_sU) * d, G, st));
    if ((r = cast_disc_weights(ws, D, pD, WD, LD, n_in, G, st, adv_pm<T>() == PM_SPLIT2)) != PIGAN_OK) return r;
  }

  const int64_t xs_gU = (int64_t)s->n_sU * d;
  const int64_t xc_g = (int64_t)S * P * d, z_g = (int64_t)S * n_z;
  const int n_s = s->n_sY + s->n_sU;
  // the Y generator's sensor locations (the trunk's: both sets)
  const float* xsG = pl.trunk ? tp<float>(ws, pl.Y.xsc) : xsY;
  const int64_t xs_gY = pl.trunk ? (int64_t)n_s * d : (int64_t)s->n_sY * d;
  for (int s0 = 0, ci = 0; s0 < S; s0 += pl.Sc, ++ci) {
    const int Sc = std::min(pl.Sc, S - s0);
    const int accum = ci > 0;
    const float* zc = z + (int64_t)s0 * n_z;
    const float* xcc = xc + (int64_t)s0 * P * d;
    const NetBuf Yc = chunk_view(pl.Y, Sc, P), Uc = chunk_view(pl.U, Sc, P);
    // generator forward passes (a critic-only step needs the sensor rows only:
    // the residual penalty is a generator term)
    const bool colloc = !s->critic_only;
    if ((r = gen_chunk_fwd<T>(ws, Yc, pY, xsG, xs_gY, xcc, xc_g, zc, z_g, d, n_z, Sc, P, G, st, colloc)) != PIGAN_OK)
      return r;
    if (!pl.trunk &&
        (r = gen_chunk_fwd<T>(ws, Uc, pU, xsU, xs_gU, xcc, xc_g, zc, z_g, d, n_z, Sc, P, G, st, colloc)) != PIGAN_OK)
      return r;
    // the trunk's head cotangents: the residual and the critic fill only
    // their own rows and streams (Y: value and first derivatives at the
    // collocation points, Y sensors; u: all streams, u sensors)
    const float* jetU = pl.trunk ? tp<float>(ws, Yc.jet2) : tp<float>(ws, Uc.jet);
    float* gbarU = pl.trunk ? tp<float>(ws, Yc.gbar2) : tp<float>(ws, Uc.gbar);
    const int64_t ju_g = pl.trunk ? Yc.R : Uc.R;
    if (pl.trunk) {
      ProfScope ps(st, "misc", 0.0, 0.0);
      HIP_TRY(launch_fill_f32(tp<float>(ws, Yc.gbar), Yc.rows, Yc.R, 0.0f, G, st));
      HIP_TRY(launch_fill_f32(gbarU, Yc.rows, Yc.R, 0.0f, G, st));
    }
    // residual and its cotangents
    if (colloc) {
      ResidArgs ra{};
      ra.jY = tp<float>(ws, Yc.jet); ra.jy_g = Yc.R; ra.offY = Yc.n_sen;
      ra.jU = jetU; ra.ju_g = ju_g; ra.offU = pl.trunk ? Yc.n_sen : Uc.n_sen;
      ra.plane = Yc.n_col; ra.M = (int64_t)Sc * P; ra.d = d;
      ra.f = f ? f + (int64_t)s0 * P : nullptr; ra.f_g = (int64_t)S * P; ra.f_const = f_const;
      ra.gY = tp<float>(ws, Yc.gbar); ra.gU = gbarU;
      ra.w_group = w_group; ra.qscale = (float)(2.0 * s->lambda_pde * ls / ((double)S * P));
      ra.part = tp<double>(ws, pl.rpart);
      ProfScope ps(st, "residual", 0.0, (double)ra.M * (3 * d + 2) * 4.0 * 2 * G);
      HIP_TRY(launch_residual(ra, G, st));
      HIP_TRY(launch_sum_partials(tp<double>(ws, pl.rpart), residual_blocks(ra.M), acc, 4, 2, G, st));
    }
    // critic forward on fake (and, in the first chunk, real) snapshots
    const int n_real = ci == 0 ? s->B_r : 0;
    const int B = Sc + n_real;
    const int64_t dact = D.Bmax * WD;
    {
      ProfScope ps(st, "misc", 0.0, 0.0);
      if (pl.trunk)   // sample s's sensor rows: [Y sensors ; u sensors], Y head then u head values
        HIP_TRY(launch_snap_fill_rows<float>(tp<float>(ws, Yc.jet), Yc.R, jetU, ju_g, s->n_sY, s->n_sU, n_s, s->n_sY,
                                             Sc, real, (int64_t)s->B_r * n_in, n_real, n_in, tp<float>(ws, D.X0),
                                             D.Bmax * D.Kp, D.Kp, G, st));
      else
        HIP_TRY(launch_snap_fill<float>(tp<float>(ws, Yc.jet), Yc.R, tp<float>(ws, Uc.jet), Uc.R, s->n_sY, s->n_sU,
                                        Sc, real, (int64_t)s->B_r * n_in, n_real, n_in, tp<float>(ws, D.X0),
                                        D.Bmax * D.Kp, D.Kp, G, st));
    }
    int cur = 0;
    if ((r = disc_pass(ws, pl, pD, WD, LD, n_in, B, Sc, n_real, S, s->B_r, w_group, ls, inv, accum, gD, nonfinite,
                       acc, G, st, &cur, pm)) != PIGAN_OK)
      return r;
    if (!s->critic_only) {
      // d(L_adv)/dF = -dL_D/dF for the fake rows -> generator sensor cotangents
      NtArgs<float> a{};
      a.X = tp<float>(ws, D.dA[cur]); a.x_g = dact; a.ldx = WD;
      a.Wm = tp<float>(ws, D.w1T); a.w_g = (int64_t)WD * D.Kp; a.ldw = WD;
      a.N = D.Kp; a.K = WD; a.pm = pm; a.seg = Seg{Sc, 0, 0};
      a.seedY = tp<float>(ws, Yc.gbar); a.sY_g = Yc.R; a.seedU = gbarU; a.sU_g = ju_g;
      a.nY = s->n_sY; a.nU = s->n_sU; a.df_sign = -1.0f;
      if (pl.trunk) {
        a.sY_ld = n_s; a.sU_ld = n_s; a.sU_off = s->n_sY;
      }
      if ((r = gemm_nt<float>(EPI_DF, 0, 0, a, G, st, "disc_bwd")) != PIGAN_OK) return r;
    }
    // critic gradient penalty on the pairs of this chunk's samples
    if (s->lambda_gp > 0.0f) {
      const int n_gp = std::min(S, s->B_r), npair = std::min(n_gp, s0 + Sc) - s0;
      const int ldY = pl.trunk ? n_s : s->n_sY, ldU = pl.trunk ? n_s : s->n_sU, offU = pl.trunk ? s->n_sY : 0;
      if (npair > 0) {
        {
          ProfScope ps(st, "gp_misc", 0.0, 0.0);
          HIP_TRY(launch_gp_mix<float>(tp<float>(ws, Yc.jet), Yc.R, jetU, ju_g, s->n_sY, s->n_sU, ldY, ldU, offU, real,
                                       (int64_t)s->B_r * n_in, gp_eps, n_gp, s0, npair, n_in, tp<float>(ws, D.X0),
                                       D.Bmax * D.Kp, D.Kp, G, st));
        }
        if ((r = critic_penalty(ws, pl, s, pD, w_group, npair, gD, inv, nonfinite, acc, G, st, pm)) != PIGAN_OK)
          return r;
      }
    }
    // generator reverse passes (not in a critic-only step)
    if (s->critic_only) continue;
    if ((r = gen_chunk_bwd<T>(ws, pl, Yc, pY, xsG, xs_gY, xcc, xc_g, zc, z_g, d, n_z, Sc, P, gY, accum, inv, nonfinite,
                              G, st)) != PIGAN_OK)
      return r;
    if (!pl.trunk && (r = gen_chunk_bwd<T>(ws, pl, Uc, pU, xsU, xs_gU, xcc, xc_g, zc, z_g, d, n_z, Sc, P, gU, accum,
                                           inv, nonfinite, G, st)) != PIGAN_OK)
      return r;
  }
  {
    ProfScope ps(st, "misc", 0.0, 0.0);
    HIP_TRY(launch_losses(acc, 4, w_group, S, s->B_r, (int64_t)S * P, s->lambda_pde, s->lambda_gp,
                          std::min(S, s->B_r), loss, gp, nonfinite, G, st));
  }
  return PIGAN_OK;
}

// Domain decomposition: one generator (a pair, or the shared trunk when
// pl.trunk: then pY is the trunk, pU and gU are unused), s->disc.n_groups
// critics (one per subdomain), each on the paper's snapshot of its subdomain
// (Y and u sensors, the generated source at free sensors and their
// coordinates).
template <class T>
static pigan_status run_hier(const pigan_step_desc* s, const StepPlan& pl, const float* pY, const float* pU,
                             const float* pD, const float* z, const float* xc, const float* xsY, const float* xsU,
                             const float* f, float f_const, const int32_t* idxY, const int32_t* idxU,
                             const int32_t* idxF, int mY, int mU, int nF, const float* real, const float* w_disc,
                             float* gY, float* gU, float* gD, float* loss, int32_t* nonfinite, void* ws,
                             hipStream_t st, const float* gp_eps, float* gp) {
  const int GD = pl.GD, d = s->d, n_z = s->n_z, P = s->P, S = s->S;
  const float ls = s->loss_scale;
  const float inv = 1.0f / ls;
  const DiscBuf& D = pl.D;
  const int WD = s->disc.width, LD = s->disc.n_hidden, n_in = s->disc.in_dim;
  const int pm = adv_pm<T>();
  double* acc = tp<double>(ws, pl.acc);
  pigan_status r;
  {
    ProfScope ps(st, "misc", 0.0, 0.0);
    HIP_TRY(launch_zero(acc, 4 * GD, nonfinite, st));
    if ((r = cast_gen_weights<T>(ws, pl.Y, pY, 1, st)) != PIGAN_OK) return r;
    if (!pl.trunk && (r = cast_gen_weights<T>(ws, pl.U, pU, 1, st)) != PIGAN_OK) return r;
    if (pl.trunk)   // the trunk sees both sensor sets: locations [Y sensors ; u sensors]
      HIP_TRY(launch_concat_rows(xsY, (int64_t)s->n_sY * d, s->n_sY, xsU, (int64_t)s->n_sU * d, s->n_sU, d,
                                 tp<float>(ws, pl.Y.xsc), (int64_t)(s->n_sY + s->n_sU) * d, 1, st));
    if ((r = cast_disc_weights(ws, D, pD, WD, LD, n_in, GD, st, adv_pm<T>() == PM_SPLIT2)) != PIGAN_OK) return r;
  }
  const int n_s = s->n_sY + s->n_sU;
  const float* xsG = pl.trunk ? tp<float>(ws, pl.Y.xsc) : xsY;
  const int64_t xs_gY = pl.trunk ? (int64_t)n_s * d : (int64_t)s->n_sY * d, xs_gU = (int64_t)s->n_sU * d;
  const int64_t xc_g = (int64_t)S * P * d, z_g = (int64_t)S * n_z;
  float* rbuf = tp<float>(ws, pl.hr);
  float* gN = tp<float>(ws, pl.hgn);
  float* dX = tp<float>(ws, pl.hdx);
  const int64_t dx_g = (int64_t)pl.Sc * D.Kp;
  for (int s0 = 0, ci = 0; s0 < S; s0 += pl.Sc, ++ci) {
    const int Sc = std::min(pl.Sc, S - s0);
    const int accum = ci > 0;
    const float* zc = z + (int64_t)s0 * n_z;
    const float* xcc = xc + (int64_t)s0 * P * d;
    const NetBuf Yc = chunk_view(pl.Y, Sc, P), Uc = chunk_view(pl.U, Sc, P);
    if ((r = gen_chunk_fwd<T>(ws, Yc, pY, xsG, xs_gY, xcc, xc_g, zc, z_g, d, n_z, Sc, P, 1, st)) != PIGAN_OK) return r;
    if (!pl.trunk &&
        (r = gen_chunk_fwd<T>(ws, Uc, pU, xsU, xs_gU, xcc, xc_g, zc, z_g, d, n_z, Sc, P, 1, st)) != PIGAN_OK)
      return r;
    // the u outputs and their cotangents: the trunk's second head, or the u network
    const float* jetU = pl.trunk ? tp<float>(ws, Yc.jet2) : tp<float>(ws, Uc.jet);
    float* gbarU = pl.trunk ? tp<float>(ws, Yc.gbar2) : tp<float>(ws, Uc.gbar);
    const int64_t rowsU = pl.trunk ? Yc.rows : Uc.rows, ju_g = pl.trunk ? Yc.R : Uc.R;
    const int64_t M = (int64_t)Sc * P;
    ResidArgs ra{};
    ra.jY = tp<float>(ws, Yc.jet); ra.jy_g = Yc.R; ra.offY = Yc.n_sen;
    ra.jU = jetU; ra.ju_g = ju_g; ra.offU = pl.trunk ? Yc.n_sen : Uc.n_sen;
    ra.plane = Yc.n_col; ra.M = M; ra.d = d;
    ra.f = f ? f + (int64_t)s0 * P : nullptr; ra.f_g = (int64_t)S * P; ra.f_const = f_const;
    {
      // the residual (its values feed the critics' free sensors) and the penalty's sum
      ProfScope ps(st, "residual", 0.0, (double)M * (3 * d + 2) * 4.0);
      ResidArgs r1 = ra;
      r1.r = rbuf; r1.r_g = M; r1.part = tp<double>(ws, pl.rpart);
      HIP_TRY(launch_residual(r1, 1, st));
      HIP_TRY(launch_sum_partials(tp<double>(ws, pl.rpart), residual_blocks(M), acc, 4, 2, 1, st));
    }
    HierSnap h{};
    h.jY = tp<float>(ws, Yc.jet); h.jU = jetU; h.nsY = s->n_sY; h.nsU = s->n_sU;
    h.ldY = pl.trunk ? n_s : s->n_sY; h.ldU = pl.trunk ? n_s : s->n_sU; h.offU = pl.trunk ? s->n_sY : 0;
    h.r = rbuf; h.f = ra.f; h.f_const = f_const; h.xc = xcc; h.P = P; h.d = d;
    h.idxY = idxY; h.idxU = idxU; h.idxF = idxF; h.mY = mY; h.mU = mU; h.nF = nF; h.n_in = n_in;
    h.bad = nonfinite;
    const int n_real = ci == 0 ? s->B_r : 0;
    const int B = Sc + n_real;
    {
      ProfScope ps(st, "misc", 0.0, 0.0);
      HIP_TRY(launch_fill_f32(tp<float>(ws, Yc.gbar), Yc.rows, Yc.R, 0.0f, 1, st));
      HIP_TRY(launch_fill_f32(gbarU, rowsU, ju_g, 0.0f, 1, st));
      HIP_TRY(launch_fill_f32(gN, M, M, 0.0f, 1, st));
      HIP_TRY(launch_hier_snap<float>(h, Sc, real, (int64_t)s->B_r * n_in, n_real, tp<float>(ws, D.X0),
                                      D.Bmax * D.Kp, D.Kp, GD, st));
    }
    int cur = 0;
    if ((r = disc_pass(ws, pl, pD, WD, LD, n_in, B, Sc, n_real, S, s->B_r, w_disc, ls, inv, accum, gD, nonfinite,
                       acc, GD, st, &cur, pm)) != PIGAN_OK)
      return r;
    if (!s->critic_only) {
      // -dL_D/dX of every critic's fake rows (all inputs), then added to the
      // generator outputs they were read from
      const int64_t dact = D.Bmax * WD;
      NtArgs<float> a{};
      a.X = tp<float>(ws, D.dA[cur]); a.x_g = dact; a.ldx = WD;
      a.Wm = tp<float>(ws, D.w1T); a.w_g = (int64_t)WD * D.Kp; a.ldw = WD;
      a.N = D.Kp; a.K = WD; a.pm = pm; a.seg = Seg{Sc, 0, 0};
      a.seedY = dX; a.sY_g = dx_g; a.sY_ld = D.Kp; a.nY = n_in; a.nU = 0; a.df_sign = -1.0f;
      if ((r = gemm_nt<float>(EPI_DF, 0, 0, a, GD, st, "disc_bwd")) != PIGAN_OK) return r;
      ProfScope ps(st, "misc", 0.0, 0.0);
      HIP_TRY(launch_hier_scatter(h, dX, dx_g, D.Kp, Sc, GD, tp<float>(ws, Yc.gbar), gbarU, gN, st));
    }
    // every critic's gradient penalty on the pairs of this chunk's samples
    // (the critics' input rows are free again: the interpolates replace them)
    if (s->lambda_gp > 0.0f) {
      const int n_gp = std::min(S, s->B_r), npair = std::min(n_gp, s0 + Sc) - s0;
      if (npair > 0) {
        {
          ProfScope ps(st, "gp_misc", 0.0, 0.0);
          HIP_TRY(launch_hier_snap<float>(h, npair, real, (int64_t)s->B_r * n_in, 0, tp<float>(ws, D.X0),
                                          D.Bmax * D.Kp, D.Kp, GD, st, gp_eps, n_gp, s0));
        }
        if ((r = critic_penalty(ws, pl, s, pD, w_disc, npair, gD, inv, nonfinite, acc, GD, st, pm)) != PIGAN_OK)
          return r;
      }
    }
    if (s->critic_only) continue;   // no generator reverse pass
    {
      // jet cotangents from the penalty and the critics' source cotangents
      ProfScope ps(st, "residual", 0.0, (double)M * (3 * d + 2) * 4.0 * 2);
      ResidArgs r2 = ra;
      r2.gY = tp<float>(ws, Yc.gbar); r2.gU = gbarU; r2.gq = gN; r2.gq_g = M;
      r2.qscale = (float)(2.0 * s->lambda_pde * ls / ((double)S * P));
      HIP_TRY(launch_residual(r2, 1, st));
    }
    if ((r = gen_chunk_bwd<T>(ws, pl, Yc, pY, xsG, xs_gY, xcc, xc_g, zc, z_g, d, n_z, Sc, P, gY, accum, inv, nonfinite,
                              1, st)) != PIGAN_OK)
      return r;
    if (!pl.trunk && (r = gen_chunk_bwd<T>(ws, pl, Uc, pU, xsU, xs_gU, xcc, xc_g, zc, z_g, d, n_z, Sc, P, gU, accum,
                                           inv, nonfinite, 1, st)) != PIGAN_OK)
      return r;
  }
  {
    ProfScope ps(st, "misc", 0.0, 0.0);
    HIP_TRY(launch_losses(acc, 4, w_disc, S, s->B_r, (int64_t)S * P, 0.0f, s->lambda_gp, std::min(S, s->B_r), loss,
                          gp, nonfinite, GD, st));
    HIP_TRY(launch_hier_pde_loss(acc, 2, s->lambda_pde, (int64_t)S * P, loss, GD, nonfinite, st));
  }
  return PIGAN_OK;
}

}  // namespace pigan

using namespace pigan;

// ===========================================================================
// C entry points
// ===========================================================================
extern "C" {

const char* pigan_last_error(void) { return g_err.c_str(); }

int64_t pigan_mlp_n_params(const pigan_mlp* net) {
  if (!net) return -1;
  MlpOff o;
  o.init(net->in_dim, net->n_hidden, net->width);
  return o.n;
}

size_t pigan_workspace_bytes(const pigan_step_desc* s) {
  if (check_step(s, true) != PIGAN_OK) return 0;   // either entry point: includes the penalty's buffers
  StepPlan pl;
  plan_step(s, choose_chunk(s), pl);
  return pl.total;
}

}  // extern "C"

static pigan_status train_step_entry(const pigan_step_desc* s, const float* pY, const float* pU, const float* pD,
                                     const float* z, const float* xc, const float* xsY, const float* xsU,
                                     const float* f, float f_const, const float* real, const float* w_group,
                                     const float* gp_eps, float* gY, float* gU, float* gD, float* loss, float* gp,
                                     int32_t* nonfinite, void* ws, size_t ws_bytes, void* stream, bool gp_entry) {
  g_err.clear();
  pigan_status st = check_step(s, gp_entry);
  if (st != PIGAN_OK) return st;
  const bool gen_out = !s->critic_only;   // the generators' gradients are outputs
  if (!pY || !pU || !pD || !z || !xc || !xsY || !xsU || !real || (gen_out && (!gY || !gU)) || !gD || !loss ||
      !nonfinite)
    return fail(PIGAN_EINVAL, "null input or output pointer");
  if (s->lambda_gp > 0.0f && !gp_eps) return fail(PIGAN_EINVAL, "lambda_gp > 0 needs gp_eps");
  if (!__builtin_isfinite(f_const)) return fail(PIGAN_EINVAL, "f_const must be finite");
  StepPlan pl;
  plan_step(s, choose_chunk(s), pl);
  if (!ws) return fail(PIGAN_EWORKSPACE, "null workspace (need %zu bytes)", pl.total);
  if (ws_bytes < pl.total) return fail(PIGAN_EWORKSPACE, "workspace has %zu bytes, need %zu", ws_bytes, pl.total);
  if ((uintptr_t)ws % 256) return fail(PIGAN_EINVAL, "workspace must be 256-byte aligned");
  hipStream_t hs = (hipStream_t)stream;
  switch (s->dt) {
    case PIGAN_FP32:
      return run_step<float>(s, pl, pY, pU, pD, z, xc, xsY, xsU, f, f_const, real, w_group, gY, gU, gD, loss,
                             nonfinite, ws, hs, gp_eps, gp);
    case PIGAN_BF16:
      return run_step<bf16>(s, pl, pY, pU, pD, z, xc, xsY, xsU, f, f_const, real, w_group, gY, gU, gD, loss,
                            nonfinite, ws, hs, gp_eps, gp);
    default:
      return run_step<f16>(s, pl, pY, pU, pD, z, xc, xsY, xsU, f, f_const, real, w_group, gY, gU, gD, loss,
                           nonfinite, ws, hs, gp_eps, gp);
  }
}

// descriptor of the domain-decomposition step as the shared step fields
// gp_name: the entry point that takes the penalty's mixing weights
static pigan_status check_hier(const pigan_hier_desc* h, pigan_step_desc* out, bool gp_entry = false,
                               const char* gp_name = "pigan_hier_step_grads_gp") {
  if (!h) return fail(PIGAN_EINVAL, "null hierarchical step descriptor");
  pigan_status st;
  if ((st = check_mlp(&h->genY, "genY")) != PIGAN_OK) return st;
  if ((st = check_mlp(&h->genU, "genU")) != PIGAN_OK) return st;
  if ((st = check_mlp(&h->disc, "disc")) != PIGAN_OK) return st;
  if ((st = check_dtype(h->dt)) != PIGAN_OK) return st;
  if (h->genY.n_groups != 1 || h->genU.n_groups != 1)
    return fail(PIGAN_EINVAL, "one generator for the whole domain: its n_groups must be 1");
  if (h->d < 1 || h->d > 3) return fail(PIGAN_EINVAL, "d=%d must be 1, 2 or 3", h->d);
  if (h->n_z < 1) return fail(PIGAN_EINVAL, "n_z=%d must be >= 1", h->n_z);
  if (h->genY.in_dim != h->d + h->n_z || h->genU.in_dim != h->d + h->n_z)
    return fail(PIGAN_EINVAL, "generator in_dim must equal d + n_z = %d", h->d + h->n_z);
  if (h->S < 1 || h->P < 1) return fail(PIGAN_EINVAL, "S=%d and P=%d must be >= 1", h->S, h->P);
  if (h->n_sY < 1 || h->n_sU < 1) return fail(PIGAN_EINVAL, "n_sY=%d and n_sU=%d must be >= 1", h->n_sY, h->n_sU);
  if (h->mY < 0 || h->mU < 0 || h->nF < 0 || h->mY + h->mU + h->nF < 1)
    return fail(PIGAN_EINVAL, "mY=%d, mU=%d, nF=%d must be >= 0 with at least one input", h->mY, h->mU, h->nF);
  if (h->disc.in_dim != h->mY + h->mU + h->nF * (1 + h->d))
    return fail(PIGAN_EINVAL, "disc in_dim=%d must equal mY + mU + nF (1 + d) = %d", h->disc.in_dim,
                h->mY + h->mU + h->nF * (1 + h->d));
  if (h->B_r < 1) return fail(PIGAN_EINVAL, "B_r=%d must be >= 1", h->B_r);
  if (h->chunk_S < 0) return fail(PIGAN_EINVAL, "chunk_S=%d must be >= 0", h->chunk_S);
  if (!(h->lambda_pde >= 0.0f) || !__builtin_isfinite(h->lambda_pde))
    return fail(PIGAN_EINVAL, "lambda_pde must be finite and >= 0");
  if (!(h->loss_scale > 0.0f) || !__builtin_isfinite(h->loss_scale))
    return fail(PIGAN_EINVAL, "loss_scale must be finite and > 0");
  if (!(h->lambda_gp >= 0.0f) || !__builtin_isfinite(h->lambda_gp))
    return fail(PIGAN_EINVAL, "lambda_gp must be finite and >= 0");
  if (!gp_entry && h->lambda_gp != 0.0f)
    return fail(PIGAN_ENOTSUP, "lambda_gp != 0 needs the per-pair mixing weights: use %s", gp_name);
  if (h->critic_only != 0 && h->critic_only != 1)
    return fail(PIGAN_EINVAL, "critic_only=%d must be 0 or 1", h->critic_only);
  pigan_step_desc s{};
  s.genY = h->genY; s.genU = h->genU; s.disc = h->disc;
  s.d = h->d; s.n_z = h->n_z; s.S = h->S; s.P = h->P; s.n_sY = h->n_sY; s.n_sU = h->n_sU; s.B_r = h->B_r;
  s.chunk_S = h->chunk_S; s.dt = h->dt; s.lambda_pde = h->lambda_pde; s.lambda_gp = h->lambda_gp;
  s.loss_scale = h->loss_scale; s.critic_only = h->critic_only;
  *out = s;
  return PIGAN_OK;
}

// the trunk step runs on the step machinery: the trunk in the Y slot (and,
// for the shape checks, the U slot), no gradient penalty
static pigan_step_desc trunk_as_step(const pigan_trunk_desc* t) {
  pigan_step_desc s{};
  s.genY = t->trunk; s.genU = t->trunk; s.disc = t->disc;
  s.d = t->d; s.n_z = t->n_z; s.S = t->S; s.P = t->P; s.n_sY = t->n_sY; s.n_sU = t->n_sU; s.B_r = t->B_r;
  s.chunk_S = t->chunk_S; s.dt = t->dt; s.lambda_pde = t->lambda_pde; s.lambda_gp = t->lambda_gp;
  s.loss_scale = t->loss_scale; s.critic_only = t->critic_only;
  return s;
}

// the hierarchical trunk step runs on the hierarchy machinery: the trunk in
// the Y slot (and, for the shape checks, the U slot)
static pigan_hier_desc hier_trunk_as_hier(const pigan_hier_trunk_desc* t) {
  pigan_hier_desc h{};
  h.genY = t->trunk; h.genU = t->trunk; h.disc = t->disc;
  h.d = t->d; h.n_z = t->n_z; h.S = t->S; h.P = t->P; h.n_sY = t->n_sY; h.n_sU = t->n_sU; h.B_r = t->B_r;
  h.chunk_S = t->chunk_S; h.mY = t->mY; h.mU = t->mU; h.nF = t->nF; h.dt = t->dt; h.lambda_pde = t->lambda_pde;
  h.loss_scale = t->loss_scale; h.lambda_gp = t->lambda_gp; h.critic_only = t->critic_only;
  return h;
}

// every hierarchical entry point: trunk selects the shared-trunk generator
// (pY is the trunk, pU and gU unused), gp_entry the entry points that take the
// penalty's mixing weights
static pigan_status hier_entry(const pigan_hier_desc* h, bool trunk, bool gp_entry, const char* gp_name,
                               const float* pY, const float* pU, const float* pD, const float* z, const float* xc,
                               const float* xsY, const float* xsU, const float* f, float f_const,
                               const int32_t* idxY, const int32_t* idxU, const int32_t* idxF, const float* real,
                               const float* w_disc, const float* gp_eps, float* gY, float* gU, float* gD,
                               float* loss, float* gp, int32_t* nonfinite, void* ws, size_t ws_bytes,
                               void* stream) {
  pigan_step_desc s;
  pigan_status st = check_hier(h, &s, gp_entry, gp_name);
  if (st != PIGAN_OK) return st;
  const bool gen_out = !s.critic_only;   // the generators' gradients are outputs
  if (!pY || (!trunk && (!pU || (gen_out && !gU))) || !pD || !z || !xc || !xsY || !xsU || !real || !w_disc ||
      (gen_out && !gY) || !gD || !loss || !nonfinite)
    return fail(PIGAN_EINVAL, "null input or output pointer");
  if ((h->mY > 0 && !idxY) || (h->mU > 0 && !idxU) || (h->nF > 0 && !idxF))
    return fail(PIGAN_EINVAL, "null sensor index list");
  if (s.lambda_gp > 0.0f && !gp_eps) return fail(PIGAN_EINVAL, "lambda_gp > 0 needs gp_eps");
  if (!__builtin_isfinite(f_const)) return fail(PIGAN_EINVAL, "f_const must be finite");
  StepPlan pl;
  plan_hier(&s, choose_chunk(&s, trunk, true), pl, trunk);
  if (!ws) return fail(PIGAN_EWORKSPACE, "null workspace (need %zu bytes)", pl.total);
  if (ws_bytes < pl.total) return fail(PIGAN_EWORKSPACE, "workspace has %zu bytes, need %zu", ws_bytes, pl.total);
  if ((uintptr_t)ws % 256) return fail(PIGAN_EINVAL, "workspace must be 256-byte aligned");
  hipStream_t hs = (hipStream_t)stream;
  if (trunk) {
    pU = nullptr;
    gU = nullptr;
  }
  switch (s.dt) {
    case PIGAN_FP32:
      return run_hier<float>(&s, pl, pY, pU, pD, z, xc, xsY, xsU, f, f_const, idxY, idxU, idxF, h->mY, h->mU, h->nF,
                             real, w_disc, gY, gU, gD, loss, nonfinite, ws, hs, gp_eps, gp);
    case PIGAN_BF16:
      return run_hier<bf16>(&s, pl, pY, pU, pD, z, xc, xsY, xsU, f, f_const, idxY, idxU, idxF, h->mY, h->mU, h->nF,
                            real, w_disc, gY, gU, gD, loss, nonfinite, ws, hs, gp_eps, gp);
    default:
      return run_hier<f16>(&s, pl, pY, pU, pD, z, xc, xsY, xsU, f, f_const, idxY, idxU, idxF, h->mY, h->mU, h->nF,
                           real, w_disc, gY, gU, gD, loss, nonfinite, ws, hs, gp_eps, gp);
  }
}

extern "C" {

pigan_status pigan_adam_update(int64_t n, float* params, const float* grads, float* m, float* v, float lr,
                               float beta1, float beta2, float eps, int32_t t, const int32_t* skip, void* stream) {
  g_err.clear();
  if (n < 0) return fail(PIGAN_EINVAL, "n=%lld must be >= 0", (long long)n);
  if (n > 0 && (!params || !grads || !m || !v)) return fail(PIGAN_EINVAL, "null parameter, gradient or moment pointer");
  if (t < 1) return fail(PIGAN_EINVAL, "t=%d must be >= 1", t);
  if (!(beta1 >= 0.0f && beta1 < 1.0f) || !(beta2 >= 0.0f && beta2 < 1.0f))
    return fail(PIGAN_EINVAL, "beta1=%g and beta2=%g must lie in [0, 1)", beta1, beta2);
  if (!__builtin_isfinite(lr) || !(eps >= 0.0f) || !__builtin_isfinite(eps))
    return fail(PIGAN_EINVAL, "lr must be finite and eps finite and >= 0");
  const float c1 = (float)(1.0 / (1.0 - std::pow((double)beta1, (double)t)));
  const float c2 = (float)(1.0 / (1.0 - std::pow((double)beta2, (double)t)));
  hipError_t e = launch_adam(n, params, grads, m, v, lr, beta1, beta2, eps, c1, c2, skip, (hipStream_t)stream);
  if (e != hipSuccess) return fail(PIGAN_EDEVICE, "adam update: %s", hipGetErrorString(e));
  return PIGAN_OK;
}

size_t pigan_hier_workspace_bytes(const pigan_hier_desc* h) {
  pigan_step_desc s;
  if (check_hier(h, &s, true) != PIGAN_OK) return 0;   // either entry point: includes the penalty's buffers
  StepPlan pl;
  plan_hier(&s, choose_chunk(&s, false, true), pl);
  return pl.total;
}

size_t pigan_hier_trunk_workspace_bytes(const pigan_hier_trunk_desc* t) {
  if (!t) return 0;
  const pigan_hier_desc h = hier_trunk_as_hier(t);
  pigan_step_desc s;
  if (check_hier(&h, &s, true) != PIGAN_OK) return 0;
  StepPlan pl;
  plan_hier(&s, choose_chunk(&s, true, true), pl, true);
  return pl.total;
}

pigan_status pigan_hier_trunk_step_grads(const pigan_hier_trunk_desc* t, const float* pT, const float* pD,
                                         const float* z, const float* xc, const float* xsY, const float* xsU,
                                         const float* f, float f_const, const int32_t* idxY, const int32_t* idxU,
                                         const int32_t* idxF, const float* real, const float* w_disc, float* gT,
                                         float* gD, float* loss, int32_t* nonfinite, void* ws, size_t ws_bytes,
                                         void* stream) {
  g_err.clear();
  if (!t) return fail(PIGAN_EINVAL, "null hierarchical trunk step descriptor");
  const pigan_hier_desc h = hier_trunk_as_hier(t);
  return hier_entry(&h, true, false, "pigan_hier_trunk_step_grads_gp", pT, nullptr, pD, z, xc, xsY, xsU, f, f_const,
                    idxY, idxU, idxF, real, w_disc, nullptr, gT, nullptr, gD, loss, nullptr, nonfinite, ws, ws_bytes,
                    stream);
}

pigan_status pigan_hier_trunk_step_grads_gp(const pigan_hier_trunk_desc* t, const float* pT, const float* pD,
                                            const float* z, const float* xc, const float* xsY, const float* xsU,
                                            const float* f, float f_const, const int32_t* idxY,
                                            const int32_t* idxU, const int32_t* idxF, const float* real,
                                            const float* w_disc, const float* gp_eps, float* gT, float* gD,
                                            float* loss, float* gp, int32_t* nonfinite, void* ws, size_t ws_bytes,
                                            void* stream) {
  g_err.clear();
  if (!t) return fail(PIGAN_EINVAL, "null hierarchical trunk step descriptor");
  const pigan_hier_desc h = hier_trunk_as_hier(t);
  return hier_entry(&h, true, true, "pigan_hier_trunk_step_grads_gp", pT, nullptr, pD, z, xc, xsY, xsU, f, f_const,
                    idxY, idxU, idxF, real, w_disc, gp_eps, gT, nullptr, gD, loss, gp, nonfinite, ws, ws_bytes,
                    stream);
}

pigan_status pigan_hier_step_grads(const pigan_hier_desc* h, const float* pY, const float* pU, const float* pD,
                                   const float* z, const float* xc, const float* xsY, const float* xsU,
                                   const float* f, float f_const, const int32_t* idxY, const int32_t* idxU,
                                   const int32_t* idxF, const float* real, const float* w_disc, float* gY, float* gU,
                                   float* gD, float* loss, int32_t* nonfinite, void* ws, size_t ws_bytes,
                                   void* stream) {
  g_err.clear();
  return hier_entry(h, false, false, "pigan_hier_step_grads_gp", pY, pU, pD, z, xc, xsY, xsU, f, f_const, idxY, idxU,
                    idxF, real, w_disc, nullptr, gY, gU, gD, loss, nullptr, nonfinite, ws, ws_bytes, stream);
}

pigan_status pigan_hier_step_grads_gp(const pigan_hier_desc* h, const float* pY, const float* pU, const float* pD,
                                      const float* z, const float* xc, const float* xsY, const float* xsU,
                                      const float* f, float f_const, const int32_t* idxY, const int32_t* idxU,
                                      const int32_t* idxF, const float* real, const float* w_disc,
                                      const float* gp_eps, float* gY, float* gU, float* gD, float* loss, float* gp,
                                      int32_t* nonfinite, void* ws, size_t ws_bytes, void* stream) {
  g_err.clear();
  return hier_entry(h, false, true, "pigan_hier_step_grads_gp", pY, pU, pD, z, xc, xsY, xsU, f, f_const, idxY, idxU,
                    idxF, real, w_disc, gp_eps, gY, gU, gD, loss, gp, nonfinite, ws, ws_bytes, stream);
}

int64_t pigan_trunk_param_count(const pigan_mlp* net) {
  if (!net || net->in_dim < 1 || net->n_hidden < 1 || net->width < 1) return 0;
  MlpOff o;
  o.init(net->in_dim, net->n_hidden, net->width, 2);
  return o.n;
}

size_t pigan_trunk_workspace_bytes(const pigan_trunk_desc* t) {
  if (!t) return 0;
  const pigan_step_desc s = trunk_as_step(t);
  if (check_step(&s, true) != PIGAN_OK) return 0;   // accounts for the penalty's buffers when lambda_gp > 0
  StepPlan pl;
  plan_step(&s, choose_chunk(&s, true), pl, true);
  return pl.total;
}

static pigan_status trunk_step_entry(const pigan_trunk_desc* t, const float* pT, const float* pD, const float* z,
                                     const float* xc, const float* xsY, const float* xsU, const float* f,
                                     float f_const, const float* real, const float* w_group, const float* gp_eps,
                                     float* gT, float* gD, float* loss, float* gp, int32_t* nonfinite, void* ws,
                                     size_t ws_bytes, void* stream, bool gp_entry) {
  g_err.clear();
  if (!t) return fail(PIGAN_EINVAL, "null trunk step descriptor");
  const pigan_step_desc s = trunk_as_step(t);
  pigan_status st = check_step(&s, gp_entry, "pigan_trunk_step_grads_gp");
  if (st != PIGAN_OK) return st;
  if (!pT || !pD || !z || !xc || !xsY || !xsU || !real || (!s.critic_only && !gT) || !gD || !loss || !nonfinite)
    return fail(PIGAN_EINVAL, "null input or output pointer");
  if (s.lambda_gp > 0.0f && !gp_eps) return fail(PIGAN_EINVAL, "lambda_gp > 0 needs gp_eps");
  if (!__builtin_isfinite(f_const)) return fail(PIGAN_EINVAL, "f_const must be finite");
  StepPlan pl;
  plan_step(&s, choose_chunk(&s, true), pl, true);
  if (!ws) return fail(PIGAN_EWORKSPACE, "null workspace (need %zu bytes)", pl.total);
  if (ws_bytes < pl.total) return fail(PIGAN_EWORKSPACE, "workspace has %zu bytes, need %zu", ws_bytes, pl.total);
  if ((uintptr_t)ws % 256) return fail(PIGAN_EINVAL, "workspace must be 256-byte aligned");
  hipStream_t hs = (hipStream_t)stream;
  switch (s.dt) {
    case PIGAN_FP32:
      return run_step<float>(&s, pl, pT, nullptr, pD, z, xc, xsY, xsU, f, f_const, real, w_group, gT, nullptr, gD,
                             loss, nonfinite, ws, hs, gp_eps, gp);
    case PIGAN_BF16:
      return run_step<bf16>(&s, pl, pT, nullptr, pD, z, xc, xsY, xsU, f, f_const, real, w_group, gT, nullptr, gD,
                            loss, nonfinite, ws, hs, gp_eps, gp);
    default:
      return run_step<f16>(&s, pl, pT, nullptr, pD, z, xc, xsY, xsU, f, f_const, real, w_group, gT, nullptr, gD,
                           loss, nonfinite, ws, hs, gp_eps, gp);
  }
}

pigan_status pigan_trunk_step_grads(const pigan_trunk_desc* t, const float* pT, const float* pD, const float* z,
                                    const float* xc, const float* xsY, const float* xsU, const float* f, float f_const,
                                    const float* real, const float* w_group, float* gT, float* gD, float* loss,
                                    int32_t* nonfinite, void* ws, size_t ws_bytes, void* stream) {
  return trunk_step_entry(t, pT, pD, z, xc, xsY, xsU, f, f_const, real, w_group, nullptr, gT, gD, loss, nullptr,
                          nonfinite, ws, ws_bytes, stream, false);
}

pigan_status pigan_trunk_step_grads_gp(const pigan_trunk_desc* t, const float* pT, const float* pD, const float* z,
                                       const float* xc, const float* xsY, const float* xsU, const float* f,
                                       float f_const, const float* real, const float* w_group, const float* gp_eps,
                                       float* gT, float* gD, float* loss, float* gp, int32_t* nonfinite, void* ws,
                                       size_t ws_bytes, void* stream) {
  return trunk_step_entry(t, pT, pD, z, xc, xsY, xsU, f, f_const, real, w_group, gp_eps, gT, gD, loss, gp,
                          nonfinite, ws, ws_bytes, stream, true);
}

pigan_status pigan_train_step_grads(const pigan_step_desc* s, const float* pY, const float* pU, const float* pD,
                                    const float* z, const float* xc, const float* xsY, const float* xsU,
                                    const float* f, float f_const, const float* real, const float* w_group,
                                    float* gY, float* gU, float* gD, float* loss, int32_t* nonfinite, void* ws,
                                    size_t ws_bytes, void* stream) {
  return train_step_entry(s, pY, pU, pD, z, xc, xsY, xsU, f, f_const, real, w_group, nullptr, gY, gU, gD, loss,
                          nullptr, nonfinite, ws, ws_bytes, stream, false);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// no-allocation entry point: the workspace is a file-scope device array.  In
// host code `scratch` names a host-side stand-in, so its device address is
// taken once per device with hipGetSymbolAddress (that device current) and
// only that address is ever passed to kernels.
// ---------------------------------------------------------------------------
static __device__ __align__(256) char scratch[PIGAN_NOALLOC_SCRATCH_BYTES];
static std::mutex g_scratch_m;
static void* g_scratch_dev[64];

static pigan_status scratch_address(void** out) {
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) return fail(PIGAN_EDEVICE, "device index %d out of range", dev);
  std::lock_guard<std::mutex> lk(g_scratch_m);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p || (uintptr_t)p % 256) return fail(PIGAN_EDEVICE, "scratch array address %p is not usable", p);
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return PIGAN_OK;
}

extern "C" {

pigan_status pigan_train_step_grads_noalloc(const pigan_step_desc* s, const float* pY, const float* pU,
                                            const float* pD, const float* z, const float* xc, const float* xsY,
                                            const float* xsU, const float* f, float f_const, const float* real,
                                            const float* w_group, float* gY, float* gU, float* gD, float* loss,
                                            int32_t* nonfinite, void* stream) {
  g_err.clear();
  pigan_status st = check_step(s, false, "pigan_train_step_grads_noalloc");
  if (st != PIGAN_OK) return st;
  StepPlan pl;
  plan_step(s, choose_chunk(s), pl);
  if (pl.total > PIGAN_NOALLOC_SCRATCH_BYTES)
    return fail(PIGAN_EWORKSPACE,
                "the step needs %zu bytes of workspace; the no-allocation entry point holds %zu (set chunk_S lower "
                "or use pigan_train_step_grads)",
                pl.total, (size_t)PIGAN_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  if ((st = scratch_address(&ws)) != PIGAN_OK) return st;
  return train_step_entry(s, pY, pU, pD, z, xc, xsY, xsU, f, f_const, real, w_group, nullptr, gY, gU, gD, loss,
                          nullptr, nonfinite, ws, pl.total, stream, false);
}

pigan_status pigan_train_step_grads_gp(const pigan_step_desc* s, const float* pY, const float* pU, const float* pD,
                                       const float* z, const float* xc, const float* xsY, const float* xsU,
                                       const float* f, float f_const, const float* real, const float* w_group,
                                       const float* gp_eps, float* gY, float* gU, float* gD, float* loss, float* gp,
                                       int32_t* nonfinite, void* ws, size_t ws_bytes, void* stream) {
  return train_step_entry(s, pY, pU, pD, z, xc, xsY, xsU, f, f_const, real, w_group, gp_eps, gY, gU, gD, loss, gp,
                          nonfinite, ws, ws_bytes, stream, true);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// generator forward
// ---------------------------------------------------------------------------
struct GenFwdPlan {
  size_t zp, h[2], wc, total;
  int64_t R;
};

static GenFwdPlan plan_gen_fwd(const pigan_mlp* net, int d, int S, int P, int order, int32_t dt) {
  GenFwdPlan p{};
  Carver cv;
  const int G = net->n_groups, W = net->width, L = net->n_hidden;
  const size_t es = esize(dt);
  const int C = 1 + order * d;
  p.R = (int64_t)C * S * P;
  p.zp = cv.take((size_t)S * W * 4 * G);
  p.h[0] = cv.take((size_t)p.R * W * es * G);
  p.h[1] = cv.take((size_t)p.R * W * es * G);
  p.wc = cv.take((size_t)std::max(L - 1, 1) * W * W * es * G * (es == 2 ? 2 : 1));   // two-term rows in 16-bit storage
  p.total = round_up((int64_t)cv.off, 256);
  return p;
}

static pigan_status check_gen_fwd(const pigan_mlp* net, int d, int S, int P, int order, int32_t dt) {
  pigan_status st = check_mlp(net, "generator");
  if (st != PIGAN_OK) return st;
  if ((st = check_dtype(dt)) != PIGAN_OK) return st;
  if (d < 1 || d > 3) return fail(PIGAN_EINVAL, "d=%d must be 1, 2 or 3", d);
  if (net->in_dim <= d) return fail(PIGAN_EINVAL, "in_dim=%d must exceed d=%d (n_z >= 1)", net->in_dim, d);
  if (S < 1 || P < 1) return fail(PIGAN_EINVAL, "S=%d and P=%d must be >= 1", S, P);
  if (order < 0 || order > 2) return fail(PIGAN_EINVAL, "order=%d must be 0, 1 or 2", order);
  return PIGAN_OK;
}

extern "C" {

size_t pigan_gen_forward_workspace(const pigan_mlp* net, int32_t d, int32_t S, int32_t P, int32_t order,
                                   int32_t dt) {
  if (check_gen_fwd(net, d, S, P, order, dt) != PIGAN_OK) return 0;
  return plan_gen_fwd(net, d, S, P, order, dt).total;
}

}  // extern "C"

template <class T>
static pigan_status run_gen_fwd(const pigan_mlp* net, const float* params, int d, const float* z, const float* x,
                                int x_shared, int S, int P, int order, float* jet, void* ws, const GenFwdPlan& p,
                                hipStream_t st) {
  const int G = net->n_groups, W = net->width, L = net->n_hidden, in_dim = net->in_dim, n_z = in_dim - d;
  MlpOff off;
  off.init(in_dim, L, W);
  const int nd1 = order >= 1 ? d : 0, nd2 = order >= 2 ? d : 0;
  const int64_t M = (int64_t)S * P;
  const int64_t actg = p.R * W;
  constexpr int tw = two_term<T>() ? 2 : 1;
  const int64_t dg = (int64_t)std::max(L - 1, 1) * W * W * tw;
  {
    ProfScope ps(st, "misc", 0.0, 0.0);
    for (int l = 2; l <= L; ++l) {
      T* dst = tp<T>(ws, p.wc) + (size_t)(l - 2) * W * W * tw;
      if constexpr (two_term<T>()) HIP_TRY(launch_cast2<T>(params + off.w[l], off.n, W, W, dst, dg, G, st));
      else HIP_TRY(launch_cast<T>(params + off.w[l], off.n, W, W, W, dst, nullptr, dg, G, st));
    }
    HIP_TRY(launch_zproj(params, off.n, in_dim, d, W, z, (int64_t)S * n_z, n_z, S, tp<float>(ws, p.zp),
                         (int64_t)S * W, G, st));
  }
  // on the resident kernel the first layer is formed inside the second
  // layer's GEMM and the output layer rides on the last one's epilogue
  const bool fuse_out = L >= 2 && nt_resident_ok((int)sizeof(T), 1 + nd1 + nd2, W, W, M, W, W);
  const int64_t x_g = x_shared ? (int64_t)P * d : M * d;
  if (!fuse_out) {
    FirstArgs<T> fa{};
    fa.p1 = params; fa.p_g = off.n; fa.in_dim = in_dim; fa.d = d; fa.W = W;
    fa.zp = tp<float>(ws, p.zp); fa.zp_g = (int64_t)S * W;
    fa.x = x; fa.x_g = x_g; fa.x_shared = x_shared ? 1 : 0; fa.Pn = P;
    fa.out_a = nullptr; fa.out_h = tp<T>(ws, p.h[0]); fa.o_g = actg; fa.ldo = W;
    fa.seg = Seg{M, 0, M};
    fa.exact = sizeof(T) == 4;
    ProfScope ps(st, "first_fwd", 2.0 * M * W * d * G, (double)M * (1 + nd1 + nd2) * W * sizeof(T) * G);
    HIP_TRY(launch_first_fwd<T>(nd1, nd2, fa, G, st));
  }
  int cur = 0;
  for (int l = 2; l <= L; ++l) {
    NtArgs<T> a{};
    a.X = tp<T>(ws, p.h[cur]); a.x_g = actg; a.ldx = W;
    a.Wm = tp<T>(ws, p.wc) + (size_t)(l - 2) * W * W * tw; a.w_g = dg; a.ldw = (int64_t)W * tw;
    a.K = W * tw; a.kx = tw == 2 ? W : 0;
    a.bias = params + off.b[l]; a.b_g = off.n;
    a.out_a = nullptr; a.out_h = tp<T>(ws, p.h[1 - cur]); a.o_g = actg; a.ldo = W;
    if (l == L && fuse_out) {
      a.out_h = nullptr;
      a.y = jet; a.y_g = p.R; a.wout = params + off.wout; a.wo_g = off.n;
    }
    if (l == 2 && fuse_out) {
      first_src(a, params, off.n, in_dim, d, tp<float>(ws, p.zp), (int64_t)S * W);
      a.fx = x; a.fx_g = x_g; a.fx_shared = x_shared ? 1 : 0; a.fPn = P;
    }
    a.N = W; a.seg = Seg{M, 0, M};
    pigan_status s1 = gemm_nt<T>(EPI_FWD, nd1, nd2, a, G, st, "gemm_fwd");
    if (s1 != PIGAN_OK) return s1;
    cur = 1 - cur;
  }
  if (!fuse_out) {
    ProfScope ps(st, "out_fwd", 2.0 * p.R * W * G, (double)p.R * W * sizeof(T) * G);
    HIP_TRY(launch_out_fwd<T>(tp<T>(ws, p.h[cur]), actg, W, p.R, M, W, params + off.wout, off.n, jet, p.R, G, st));
  }
  return PIGAN_OK;
}

extern "C" {

pigan_status pigan_gen_forward(const pigan_mlp* net, const float* params, int32_t d, const float* z, const float* x,
                               int32_t x_shared, int32_t S, int32_t P, int32_t order, int32_t dt, float* jet,
                               void* ws, size_t ws_bytes, void* stream) {
  g_err.clear();
  pigan_status st = check_gen_fwd(net, d, S, P, order, dt);
  if (st != PIGAN_OK) return st;
  if (!params || !z || !x || !jet) return fail(PIGAN_EINVAL, "null input or output pointer");
  GenFwdPlan p = plan_gen_fwd(net, d, S, P, order, dt);
  if (!ws) return fail(PIGAN_EWORKSPACE, "null workspace (need %zu bytes)", p.total);
  if (ws_bytes < p.total) return fail(PIGAN_EWORKSPACE, "workspace has %zu bytes, need %zu", ws_bytes, p.total);
  if ((uintptr_t)ws % 256) return fail(PIGAN_EINVAL, "workspace must be 256-byte aligned");
  hipStream_t hs = (hipStream_t)stream;
  switch (dt) {
    case PIGAN_FP32: return run_gen_fwd<float>(net, params, d, z, x, x_shared, S, P, order, jet, ws, p, hs);
    case PIGAN_BF16: return run_gen_fwd<bf16>(net, params, d, z, x, x_shared, S, P, order, jet, ws, p, hs);
    default: return run_gen_fwd<f16>(net, params, d, z, x, x_shared, S, P, order, jet, ws, p, hs);
  }
}

// ---------------------------------------------------------------------------
// residual
// ---------------------------------------------------------------------------
pigan_status pigan_pde_residual(int32_t d, int32_t G, int64_t M, const float* jetY, const float* jetU,
                                const float* f, float f_const, float* r, void* stream) {
  g_err.clear();
  if (d < 1 || d > 3) return fail(PIGAN_EINVAL, "d=%d must be 1, 2 or 3", d);
  if (G < 1 || G > 65535) return fail(PIGAN_EINVAL, "G=%d out of [1,65535]", G);
  if (M < 1) return fail(PIGAN_EINVAL, "M=%lld must be >= 1", (long long)M);
  if (!jetY || !jetU || !r) return fail(PIGAN_EINVAL, "null input or output pointer");
  if (!__builtin_isfinite(f_const)) return fail(PIGAN_EINVAL, "f_const must be finite");
  ResidArgs ra{};
  ra.jY = jetY; ra.jy_g = (1 + d) * M; ra.offY = 0;
  ra.jU = jetU; ra.ju_g = (1 + 2 * d) * M; ra.offU = 0;
  ra.plane = M; ra.M = M; ra.d = d;
  ra.f = f; ra.f_g = M; ra.f_const = f_const;
  ra.r = r; ra.r_g = M;
  hipStream_t hs = (hipStream_t)stream;
  ProfScope ps(hs, "residual", 0.0, (double)M * (3 * d + 3) * 4.0 * G);
  HIP_TRY(launch_residual(ra, G, hs));
  return PIGAN_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// discriminator forward
// ---------------------------------------------------------------------------
struct DiscFwdPlan {
  size_t X0, h[2], w1, wc, total;
  int Kp;
};

// the critic runs in fp32 storage in every mode (split products)
static DiscFwdPlan plan_disc_fwd(const pigan_mlp* net, int B, int32_t dt) {
  DiscFwdPlan p{};
  Carver cv;
  const int G = net->n_groups, W = net->width, L = net->n_hidden;
  const size_t es = 4;
  (void)dt;
  p.Kp = (int)round_up(net->in_dim, 32);
  p.X0 = cv.take((size_t)B * p.Kp * es * G);
  p.h[0] = cv.take((size_t)B * W * es * G);
  p.h[1] = cv.take((size_t)B * W * es * G);
  p.w1 = cv.take((size_t)W * p.Kp * es * G);
  p.wc = cv.take((size_t)std::max(L - 1, 1) * W * W * es * G);
  p.total = round_up((int64_t)cv.off, 256);
  return p;
}

extern "C" {

size_t pigan_disc_forward_workspace(const pigan_mlp* net, int32_t B, int32_t dt) {
  if (check_mlp(net, "disc") != PIGAN_OK || check_dtype(dt) != PIGAN_OK || B < 1) return 0;
  return plan_disc_fwd(net, B, dt).total;
}

}  // extern "C"

template <class T>
static pigan_status run_disc_fwd(const pigan_mlp* net, const float* params, const float* snap, int B, float* score,
                                 void* ws, const DiscFwdPlan& p, hipStream_t st) {
  const int G = net->n_groups, W = net->width, L = net->n_hidden, n_in = net->in_dim;
  MlpOff off;
  off.init(n_in, L, W);
  const int64_t actg = (int64_t)B * W;
  {
    ProfScope ps(st, "misc", 0.0, 0.0);
    // weight copies (pre-split for the split products)
    auto cast = [&](const float* src, int N, int K, int Kp, float* dst, int64_t d_g) {
      return adv_pm<T>() == PM_SPLIT2 ? launch_cast_pair(src, off.n, N, K, Kp, dst, nullptr, d_g, G, st)
                                      : launch_cast<float>(src, off.n, N, K, Kp, dst, nullptr, d_g, G, st);
    };
    HIP_TRY(cast(params + off.w[1], W, n_in, p.Kp, tp<float>(ws, p.w1), (int64_t)W * p.Kp));
    const int64_t dg = (int64_t)std::max(L - 1, 1) * W * W;
    for (int l = 2; l <= L; ++l)
      HIP_TRY(cast(params + off.w[l], W, W, W, tp<float>(ws, p.wc) + (size_t)(l - 2) * W * W, dg));
    HIP_TRY(launch_snap_fill<float>(nullptr, 0, nullptr, 0, 0, 0, 0, snap, (int64_t)B * n_in, B, n_in,
                                    tp<float>(ws, p.X0), (int64_t)B * p.Kp, p.Kp, G, st));
  }
  // layer l writes h[(l - 1) % 2]
  for (int l = 1; l <= L; ++l) {
    NtArgs<float> a{};
    if (l == 1) {
      a.X = tp<float>(ws, p.X0); a.x_g = (int64_t)B * p.Kp; a.ldx = p.Kp;
      a.Wm = tp<float>(ws, p.w1); a.w_g = (int64_t)W * p.Kp; a.ldw = p.Kp; a.K = p.Kp;
    } else {
      a.X = tp<float>(ws, p.h[(l - 2) % 2]); a.x_g = actg; a.ldx = W;
      a.Wm = tp<float>(ws, p.wc) + (size_t)(l - 2) * W * W; a.w_g = (int64_t)std::max(L - 1, 1) * W * W; a.ldw = W;
      a.K = W;
    }
    a.bias = params + off.b[l]; a.b_g = off.n;
    a.out_a = nullptr; a.out_h = tp<float>(ws, p.h[(l - 1) % 2]); a.o_g = actg; a.ldo = W;
    a.N = W; a.pm = adv_pm<T>(); a.seg = Seg{B, 0, 0};
    pigan_status s1 = gemm_nt<float>(EPI_FWD, 0, 0, a, G, st, "disc_fwd");
    if (s1 != PIGAN_OK) return s1;
  }
  const int cur = (L - 1) % 2;
  {
    ProfScope ps(st, "out_fwd", 2.0 * B * W * G, (double)B * W * 4 * G);
    HIP_TRY(launch_out_fwd<float>(tp<float>(ws, p.h[cur]), actg, W, B, B, W, params + off.wout, off.n, score, B, G,
                                  st));
  }
  return PIGAN_OK;
}

extern "C" {

pigan_status pigan_disc_forward(const pigan_mlp* net, const float* params, const float* snap, int32_t B,
                                int32_t dt, float* score, void* ws, size_t ws_bytes, void* stream) {
  g_err.clear();
  pigan_status st = check_mlp(net, "disc");
  if (st != PIGAN_OK) return st;
  if ((st = check_dtype(dt)) != PIGAN_OK) return st;
  if (B < 1) return fail(PIGAN_EINVAL, "B=%d must be >= 1", B);
  if (!params || !snap || !score) return fail(PIGAN_EINVAL, "null input or output pointer");
  DiscFwdPlan p = plan_disc_fwd(net, B, dt);
  if (!ws) return fail(PIGAN_EWORKSPACE, "null workspace (need %zu bytes)", p.total);
  if (ws_bytes < p.total) return fail(PIGAN_EWORKSPACE, "workspace has %zu bytes, need %zu", ws_bytes, p.total);
  if ((uintptr_t)ws % 256) return fail(PIGAN_EINVAL, "workspace must be 256-byte aligned");
  hipStream_t hs = (hipStream_t)stream;
  switch (dt) {
    case PIGAN_FP32: return run_disc_fwd<float>(net, params, snap, B, score, ws, p, hs);
    case PIGAN_BF16: return run_disc_fwd<bf16>(net, params, snap, B, score, ws, p, hs);
    default: return run_disc_fwd<f16>(net, params, snap, B, score, ws, p, hs);
  }
}

// ---------------------------------------------------------------------------
// profiling
// ---------------------------------------------------------------------------
pigan_status pigan_profile_enable(int32_t on) {
  std::lock_guard<std::mutex> lk(g_pm);
  g_prof = on != 0;
  return PIGAN_OK;
}

pigan_status pigan_profile_read(pigan_kernel_stat* out, int32_t max_entries, int32_t* n_entries) {
  g_err.clear();
  if (!n_entries || (max_entries > 0 && !out)) return fail(PIGAN_EINVAL, "null output");
  std::lock_guard<std::mutex> lk(g_pm);
  std::vector<pigan_kernel_stat> agg;
  for (auto& r : g_recs) {
    float ms = 0.0f;
    if (r.a && r.b) {
      hipError_t e = hipEventElapsedTime(&ms, r.a, r.b);
      if (e != hipSuccess) ms = 0.0f;
    }
    auto it = std::find_if(agg.begin(), agg.end(), [&](const pigan_kernel_stat& k) { return r.name == k.name; });
    if (it == agg.end()) {
      pigan_kernel_stat k{};
      snprintf(k.name, sizeof k.name, "%s", r.name.c_str());
      agg.push_back(k);
      it = agg.end() - 1;
    }
    it->launches += 1;
    it->total_ms += ms;
    it->flops += r.flops;
    it->bytes += r.bytes;
    if (r.a) g_pool.push_back(r.a);
    if (r.b) g_pool.push_back(r.b);
  }
  g_recs.clear();
  const int n = (int)agg.size();
  for (int i = 0; i < n && i < max_entries; ++i) out[i] = agg[i];
  *n_entries = n;
  return PIGAN_OK;
}

}  // extern "C"
