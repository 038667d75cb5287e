// C-ABI of the GMC boundary operator: context, validation, workspace plan and
// the launch sequence of one call (Algorithm 1, steps 2-6):
//   message clients -> appearance/spatial banks -> selection rounds ->
//   assignment -> transport + compaction.
// Nothing here synchronises the device; every launch goes to the context
// stream.  The workspace is one allocation made in gmc_init.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <vector>

#include "gmc.h"
#include "gmc_internal.h"
#include "gmc_kernels.h"
#include "gmc_path.h"

using namespace gmc;

namespace {

struct Capacity {
  int B, N, T, K, I, hq, hr, mv, m, ldM, pool_cap, bmax, ldK, rank;
  int cert_rounds;   // selection rounds the certificate buffers hold
  bool bounded_possible;
};

struct Context {
  gmc_config cfg{};
  Params pr{};
  Capacity cap{};
  Ws ws{};
  void* mem = nullptr;
  size_t bytes = 0;
  hipStream_t stream = nullptr;
  // internal side stream for the bank kernels (default priority); it starts
  // each call behind a device gate on the row-norm blocks' call tags (one
  // image) or an event, and joins the caller's stream through a device flag
  // (an event without text queries)
  hipStream_t side = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  int call_tag = 0;   // last call number handed to the row-norm blocks
  int device = 0;
  int diag = 0;       // GMC_DIAG_* flags for the next calls
  // the last pruning call: its stream (a call on another stream waits for it
  // through `xfer`), its shape and what it recorded
  hipStream_t last_stream = nullptr;
  // the stream of the last call of any kind that used the workspace (a
  // pruning call or an audit, whose scratch lives in the client matrix)
  hipStream_t order_stream = nullptr;
  hipEvent_t xfer = nullptr;
  bool has_call = false, last_identity = false, last_cert = false;
  Shape last{};
};

std::mutex g_mu;
Context* g_ctx = nullptr;
char g_err[512] = "";

// Stage timer: events recorded on the op stream around each stage's launches.
struct Span {
  int stage;
  hipEvent_t a, b;
};
struct Timer {
  bool on = false;
  std::vector<hipEvent_t> pool;
  size_t used = 0;
  std::vector<Span> spans;
  hipEvent_t open[kNumStages] = {};
  hipEvent_t take() {
    if (used == pool.size()) {
      hipEvent_t e = nullptr;
      if (hipEventCreate(&e) != hipSuccess) return nullptr;
      pool.push_back(e);
    }
    return pool[used++];
  }
  void release() {
    for (hipEvent_t e : pool) (void)hipEventDestroy(e);
    pool.clear();
    spans.clear();
    used = 0;
  }
};
Timer g_timer;

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}


long long round_up(long long x, long long a) { return (x + a - 1) / a * a; }
long long cdiv(long long x, long long a) { return (x + a - 1) / a; }

int app_rows(const gmc_config& c, int n) {
  return n > c.bounded_threshold_n ? std::min(c.app_max_clients, n) : n;
}

Params make_params(const gmc_config& c) {
  Params p{};
  p.lambda_mass = c.lambda_mass; p.eps_mass = c.eps_mass; p.beta_msg = c.beta_msg;
  p.beta_app = c.beta_app; p.beta_spa = c.beta_spa; p.tau_v = c.tau_v; p.tau_s = c.tau_s;
  p.tau_r = c.tau_r; p.resp_eps = c.resp_eps; p.spatial_w = c.spatial_w; p.gate_t = c.gate_t;
  p.gate_p = c.gate_p; p.amb_margin = c.amb_margin; p.amb_p = c.amb_p; p.g_form = c.g_form;
  p.pop_strength = c.pop_strength; p.tau_j = c.tau_j; p.max_head_clusters = c.max_head_clusters;
  p.disp_eps = c.disp_eps; p.terminal_q_weight = c.terminal_q_weight; p.rms_eps = c.rms_eps;
  p.norm_eps = c.norm_eps; p.restore_eps = c.restore_eps; p.pool_mult = c.pool_mult;
  p.probe_bias = c.value_probe_bias;
  p.beta_view[0] = c.beta_msg;   // one view; calls with historical views set their own masses
  return p;
}

int validate_config(const gmc_config* c) {
  if (!c) return fail(GMC_ERR_ARG, "gmc_init: cfg is NULL");
  if (c->d <= 0 || c->d % 64 != 0) return fail(GMC_ERR_ARG, "d=%d must be a positive multiple of 64", c->d);
  if (c->d > 256 * 8 * 8) return fail(GMC_ERR_ARG, "d=%d exceeds 16384", c->d);
  if (c->n_q_heads < 1 || c->n_q_heads > kMaxHeads)
    return fail(GMC_ERR_ARG, "n_q_heads=%d must be in [1, %d]", c->n_q_heads, kMaxHeads);
  if (c->n_kv_heads < 1 || c->n_q_heads % c->n_kv_heads != 0)
    return fail(GMC_ERR_ARG, "n_kv_heads=%d must divide n_q_heads=%d", c->n_kv_heads, c->n_q_heads);
  if (c->head_dim < 32 || c->head_dim > 256 || c->head_dim % 32 != 0)
    return fail(GMC_ERR_ARG, "head_dim=%d must be a multiple of 32 in [32, 256]", c->head_dim);
  if (c->probe_rank < 1 || c->probe_rank > kMaxProbe)
    return fail(GMC_ERR_ARG, "probe_rank=%d must be in [1, %d]", c->probe_rank, kMaxProbe);
  if (c->dtype != GMC_F32 && c->dtype != GMC_BF16) return fail(GMC_ERR_ARG, "dtype=%d unknown", c->dtype);
  if (c->max_batch < 1) return fail(GMC_ERR_ARG, "max_batch=%d must be >= 1", c->max_batch);
  if (c->max_n < 1 || c->max_n > kMaxN) return fail(GMC_ERR_ARG, "max_n=%d must be in [1, %d]", c->max_n, kMaxN);
  if (c->max_t < 0) return fail(GMC_ERR_ARG, "max_t=%d must be >= 0", c->max_t);
  if (c->max_k < 0 || c->max_k > c->max_n) return fail(GMC_ERR_ARG, "max_k=%d must be in [0, max_n]", c->max_k);
  if (!c->value_probe) return fail(GMC_ERR_ARG, "value_probe is NULL");
  if (c->landmarks < 1 || c->landmarks > 64) return fail(GMC_ERR_ARG, "landmarks=%d out of [1, 64]", c->landmarks);
  if (c->batch_b < 1 || c->batch_b_bounded < 1 || c->pool_mult < 1)
    return fail(GMC_ERR_ARG, "batch sizes and pool_mult must be >= 1");
  if (c->batch_b > 1024 || c->batch_b_bounded > 1024)
    return fail(GMC_ERR_ARG, "batch sizes must be <= 1024");
  if (static_cast<long long>(c->pool_mult) * std::max(c->batch_b, c->batch_b_bounded) > 2048)
    return fail(GMC_ERR_ARG, "pool_mult * batch must be <= 2048");
  if (c->max_head_clusters < 1) return fail(GMC_ERR_ARG, "max_head_clusters must be >= 1");
  if (!(c->tau_v > 0 && c->tau_s > 0 && c->tau_r > 0 && c->gate_t > 0 && c->amb_margin > 0))
    return fail(GMC_ERR_ARG, "temperatures and gate scales must be positive");
  if (c->g_form != 0 && c->g_form != 1) return fail(GMC_ERR_ARG, "g_form=%d unknown", c->g_form);
  if (c->bounded_threshold_n < 1) return fail(GMC_ERR_ARG, "bounded_threshold_n must be >= 1");
  if (c->max_hist_views < 0 || c->max_hist_views > GMC_MAX_HIST_VIEWS)
    return fail(GMC_ERR_ARG, "max_hist_views=%d must be in [0, %d]", c->max_hist_views, GMC_MAX_HIST_VIEWS);
  if (c->max_hist_views > 0 && !c->value_probe_hist)
    return fail(GMC_ERR_ARG, "value_probe_hist is NULL but max_hist_views=%d", c->max_hist_views);
  if (!(c->hist_mass >= 0.f && c->hist_mass <= 1.f))
    return fail(GMC_ERR_ARG, "hist_mass must be in [0, 1]");
  if (c->max_images < 0 || c->max_images > GMC_MAX_IMAGES)
    return fail(GMC_ERR_ARG, "max_images=%d must be in [0, %d]", c->max_images, GMC_MAX_IMAGES);
  if (c->max_n > c->bounded_threshold_n) {
    if (!c->app_projection) return fail(GMC_ERR_ARG, "app_projection is NULL but max_n exceeds the bounded threshold");
    if (c->app_rank < 64 || c->app_rank % 64 != 0 || c->app_rank > 1024)
      return fail(GMC_ERR_ARG, "app_rank=%d must be a multiple of 64 in [64, 1024]", c->app_rank);
    if (c->app_max_clients < 1) return fail(GMC_ERR_ARG, "app_max_clients must be >= 1");
  }
  return GMC_OK;
}

// Workspace plan: per-problem strides from the capacities.
struct Plan {
  Capacity cap;
  long long s_n, s_z, s_zp, s_sig, s_ell, s_E, s_m, s_apart, s_gpart, s_e2, s_om, s_eb, s_pc, s_bd, s_y, s_cl,
      s_cov, s_sel, s_ord, s_pool, s_spart, s_bat, s_slot, s_sup, s_cos, s_del, s_ftag, s_gate,
      s_pi, s_st, s_keys, s_u, s_cnt, s_rstat, s_lstat, s_tu, s_ts, s_tc, s_lpart, s_lcnt;
  long long s_gpart1, s_n2h, s_img, s_imgcnt;
  long long s_cgain, s_cscore, s_cpool, s_cbat, s_cpart, s_cert, s_dstat;
};

Plan make_plan(const gmc_config& c) {
  Plan pl{};
  Capacity& k = pl.cap;
  k.B = c.max_batch;
  k.N = c.max_n;
  k.T = c.max_t;
  k.K = c.max_k > 0 ? c.max_k : c.max_n;
  k.hq = c.n_q_heads;
  k.hr = c.n_q_heads * c.probe_rank;
  k.bounded_possible = c.max_n > c.bounded_threshold_n;
  k.mv = std::max(std::min(c.max_n, c.bounded_threshold_n),
                  k.bounded_possible ? std::min(c.app_max_clients, c.max_n) : 0);
  k.I = std::max(1, c.max_images);
  k.m = (1 + c.max_hist_views) * k.hq * k.T + k.mv + c.landmarks * c.landmarks * k.I;
  k.ldM = static_cast<int>(round_up(k.m, 4));
  k.bmax = std::max(c.batch_b, k.bounded_possible ? c.batch_b_bounded : 0);
  k.pool_cap = c.pool_mult * k.bmax;
  k.ldK = static_cast<int>(round_up(k.K, 4));
  k.rank = k.bounded_possible ? c.app_rank : 0;
  const long long npairs = static_cast<long long>(k.hq) * (k.hq + 1) / 2;
  pl.s_n = k.N;
  pl.s_z = static_cast<long long>(k.N) * k.hr;
  pl.s_zp = kProbeSplit * pl.s_z;
  pl.s_lpart = 4LL * kLogitSplit * k.hq * std::max(k.T, 1);
  pl.s_lcnt = cdiv(static_cast<long long>(c.n_q_heads / c.n_kv_heads) * std::max(k.T, 1), 16) * c.n_kv_heads;
  pl.s_sig = kMaxHeads;
  pl.s_ell = static_cast<long long>(k.hq) * k.N;
  pl.s_E = static_cast<long long>(k.N) * k.ldM;
  pl.s_m = k.ldM;
  pl.s_apart = cdiv(k.N, k.bounded_possible ? kAppBoundedTile : 64) * k.mv;
  pl.s_gpart1 = std::max(cdiv(k.N, kHeadTok) * round_up(npairs, 4), cdiv(k.N, 64) * k.hq);
  pl.s_gpart = (1 + c.max_hist_views) * pl.s_gpart1;
  pl.s_n2h = c.max_hist_views > 0 ? k.N : 1;
  pl.s_e2 = static_cast<long long>(k.hq) * k.N;
  pl.s_om = kMaxHeads;
  pl.s_eb = k.N;
  pl.s_pc = 2LL * k.N;
  pl.s_bd = 4;
  pl.s_y = static_cast<long long>(k.N) * k.rank;
  pl.s_cl = k.mv;
  pl.s_cov = k.ldM;
  pl.s_sel = k.N;
  pl.s_ord = k.N;
  pl.s_pool = k.pool_cap;
  pl.s_spart = 2 * 64 * cdiv(k.ldM, 64);
  pl.s_bat = k.bmax;
  pl.s_slot = k.N;
  pl.s_sup = k.N;
  pl.s_cos = static_cast<long long>(k.N) * k.ldK;
  pl.s_del = k.N;
  pl.s_ftag = cdiv(k.N, 4);
  pl.s_gate = 4;
  pl.s_pi = k.N;
  pl.s_st = kStats;
  pl.s_keys = k.N;
  pl.s_u = k.N;
  pl.s_cnt = kCounters;
  pl.s_rstat = 3LL * k.ldM;
  pl.s_lstat = static_cast<long long>(c.landmarks) * c.landmarks * k.I;
  pl.s_img = k.N;
  pl.s_imgcnt = kMaxImages;
  pl.s_tu = 2LL * k.N;
  pl.s_ts = 2 * 64 * cdiv(k.ldM, 64) + 2 * 64;   // chunk partials, then the published pool
  pl.s_tc = 2LL * (k.ldM + kMaxPersist);
  // certificate buffers: rounds of the smallest batch size, at most
  // kCertMaxRounds
  k.cert_rounds = static_cast<int>(std::min<long long>(
      kCertMaxRounds, cdiv(k.K, std::max(1, std::min(c.batch_b, k.bounded_possible ? c.batch_b_bounded : c.batch_b)))));
  pl.s_cgain = static_cast<long long>(k.cert_rounds) * k.N;
  pl.s_cscore = static_cast<long long>(k.cert_rounds) * k.pool_cap;
  pl.s_cpool = pl.s_cscore;
  pl.s_cbat = static_cast<long long>(k.cert_rounds) * k.bmax;
  pl.s_cpart = static_cast<long long>(k.cert_rounds) * cdiv(k.ldM, 256);
  pl.s_cert = static_cast<long long>(k.cert_rounds) * kCertFields + 4;
  pl.s_dstat = kStats;
  return pl;
}

// Carve the allocation; returns total bytes when base is nullptr.
size_t carve(const Plan& pl, char* base, Ws* ws) {
  size_t off = 0;
  const long long B = pl.cap.B;
  auto take = [&](long long per_problem, size_t esz) -> char* {
    off = round_up(off, 256);
    char* p = base ? base + off : nullptr;
    off += static_cast<size_t>(std::max<long long>(per_problem, 1) * B) * esz;
    return p;
  };
#define F(name) ws->name = reinterpret_cast<float*>(take(pl.s_##name, 4)); ws->s_##name = pl.s_##name
#define I(name) ws->name = reinterpret_cast<int*>(take(pl.s_##name, 4)); ws->s_##name = pl.s_##name
  ws->n2 = reinterpret_cast<float*>(take(pl.s_n, 4)); ws->s_n = pl.s_n;
  F(z); F(zp); F(lpart); I(lcnt); F(sig); F(ell); F(E);
  ws->alpha = reinterpret_cast<float*>(take(pl.s_m, 4)); ws->s_m = pl.s_m;
  ws->peak = reinterpret_cast<float*>(take(pl.s_m, 4));
  ws->rowsum = reinterpret_cast<float*>(take(pl.s_m, 4));
  ws->apart_sum = reinterpret_cast<float*>(take(pl.s_apart, 4));
  ws->apart_max = reinterpret_cast<float*>(take(pl.s_apart, 4)); ws->s_apart = pl.s_apart;
  F(gpart); F(e2); F(n2h); I(img); I(imgcnt);
  ws->s_gpart1 = pl.s_gpart1;
  ws->omega = reinterpret_cast<float*>(take(pl.s_om, 4)); ws->s_om = pl.s_om;
  ws->ebar = reinterpret_cast<float*>(take(pl.s_eb, 4)); ws->s_eb = pl.s_eb;
  F(pc);
  ws->bounds = reinterpret_cast<float*>(take(pl.s_bd, 4)); ws->s_bd = pl.s_bd;
  F(y);
  ws->clients = reinterpret_cast<int*>(take(pl.s_cl, 4)); ws->s_cl = pl.s_cl;
  F(cov);
  I(sel);
  ws->order = reinterpret_cast<int*>(take(pl.s_ord, 4)); ws->s_ord = pl.s_ord;
  I(pool); F(spart);
  ws->batch = reinterpret_cast<int*>(take(pl.s_bat, 4)); ws->s_bat = pl.s_bat;
  I(slot); I(sup);
  ws->cosb = reinterpret_cast<float*>(take(pl.s_cos, 4)); ws->s_cos = pl.s_cos;
  ws->delta = reinterpret_cast<float*>(take(pl.s_del, 4)); ws->s_del = pl.s_del;
  I(ftag);
  ws->gate = reinterpret_cast<float*>(take(pl.s_gate, 4)); ws->s_gate = pl.s_gate;
  I(pi);
  ws->stats = reinterpret_cast<float*>(take(pl.s_st, 4)); ws->s_st = pl.s_st;
  ws->keys = reinterpret_cast<uint32_t*>(take(pl.s_keys, 4)); ws->s_keys = pl.s_keys;
  ws->u = reinterpret_cast<float*>(take(pl.s_u, 4)); ws->s_u = pl.s_u;
  ws->cnt = reinterpret_cast<int*>(take(pl.s_cnt, 4)); ws->s_cnt = pl.s_cnt;
  ws->tu = reinterpret_cast<unsigned long long*>(take(pl.s_tu, 8)); ws->s_tu = pl.s_tu;
  ws->ts = reinterpret_cast<unsigned long long*>(take(pl.s_ts, 8)); ws->s_ts = pl.s_ts;
  ws->tc = reinterpret_cast<unsigned long long*>(take(pl.s_tc, 8)); ws->s_tc = pl.s_tc;
  F(rstat); F(lstat);
  ws->cert_rounds = pl.cap.cert_rounds;
  F(cgain); F(cscore); I(cpool); I(cbat); F(cpart); F(cert); F(dstat);
#undef F
#undef I
  return round_up(off, 256);
}

}  // namespace

namespace gmc {
int set_error(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

int check_config(const gmc_config* cfg) { return validate_config(cfg); }

Params params_of(const gmc_config& cfg) { return make_params(cfg); }

size_t carve_workspace(const gmc_config& cfg, char* base, Ws* ws) { return carve(make_plan(cfg), base, ws); }

void timer_mark(int stage, bool begin, hipStream_t st) {
  if (!g_timer.on || stage < 0 || stage >= kNumStages) return;
  hipEvent_t e = g_timer.take();
  if (!e) return;
  (void)hipEventRecord(e, st);
  if (begin) {
    g_timer.open[stage] = e;
  } else if (g_timer.open[stage]) {
    g_timer.spans.push_back(Span{stage, g_timer.open[stage], e});
    g_timer.open[stage] = nullptr;
  }
}
}  // namespace gmc

extern "C" {

void gmc_config_default(gmc_config* c) {
  if (!c) return;
  std::memset(c, 0, sizeof(*c));
  c->probe_rank = 4;
  c->dtype = GMC_BF16;
  c->max_batch = 1;
  c->lambda_mass = 1.0f;
  c->eps_mass = 1e-8f;
  c->beta_msg = 1.0f;
  c->beta_app = 0.5f;
  c->beta_spa = 0.25f;
  c->tau_v = 0.2f;
  c->tau_s = 0.02f;
  c->landmarks = 16;
  c->batch_b = 16;
  c->pool_mult = 4;
  c->tau_r = 0.1f;
  c->resp_eps = 1e-30f;
  c->spatial_w = 0.5f;
  c->gate_t = 0.08f;
  c->gate_p = 8.0f;
  c->amb_margin = 0.05f;
  c->amb_p = 8.0f;
  c->g_form = 0;
  c->pop_strength = 0.5f;
  c->tau_j = 1.0f;
  c->max_head_clusters = 4;
  c->disp_eps = 0.05f;
  c->terminal_q_weight = 2.0f;
  c->rms_eps = 1e-6f;
  c->norm_eps = 1e-12f;
  c->restore_eps = 1e-6f;
  c->bounded_threshold_n = 4096;
  c->app_rank = 128;
  c->app_max_clients = 4096;
  c->batch_b_bounded = 512;
  c->max_hist_views = 0;
  c->hist_mass = 0.5f;
  c->max_images = 1;
}

void gmc_free(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_timer.on = false;
  g_timer.release();
  if (!g_ctx) return;
  (void)hipSetDevice(g_ctx->device);
  if (g_ctx->side) {
    (void)hipStreamSynchronize(g_ctx->side);
    (void)hipStreamDestroy(g_ctx->side);
  }
  if (g_ctx->fork) (void)hipEventDestroy(g_ctx->fork);
  if (g_ctx->join) (void)hipEventDestroy(g_ctx->join);
  if (g_ctx->xfer) (void)hipEventDestroy(g_ctx->xfer);
  if (g_ctx->mem) (void)hipFree(g_ctx->mem);
  delete g_ctx;
  g_ctx = nullptr;
}

int gmc_init(const gmc_config* cfg) {
  int rc = validate_config(cfg);
  if (rc != GMC_OK) return rc;
  gmc_free();
  std::lock_guard<std::mutex> lk(g_mu);
  Context* ctx = new Context();
  ctx->cfg = *cfg;
  if (ctx->cfg.max_k == 0) ctx->cfg.max_k = ctx->cfg.max_n;
  if (ctx->cfg.max_images == 0) ctx->cfg.max_images = 1;
  ctx->pr = make_params(ctx->cfg);
  Plan pl = make_plan(ctx->cfg);
  ctx->cap = pl.cap;
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) {
    delete ctx;
    return fail(GMC_ERR_HIP, "gmc_init: no HIP device (%s)", hipGetErrorString(err));
  }
  ctx->device = dev;
  Ws tmp{};
  const size_t bytes = carve(pl, nullptr, &tmp);
  err = hipMalloc(&ctx->mem, bytes);
  if (err != hipSuccess) {
    delete ctx;
    return fail(GMC_ERR_HIP, "gmc_init: hipMalloc(%zu) failed (%s)", bytes, hipGetErrorString(err));
  }
  ctx->bytes = bytes;
  carve(pl, static_cast<char*>(ctx->mem), &ctx->ws);
  err = hipMemset(ctx->mem, 0, bytes);
  if (err == hipSuccess) err = hipDeviceSynchronize();
  if (err != hipSuccess) {
    (void)hipFree(ctx->mem);
    delete ctx;
    return fail(GMC_ERR_HIP, "gmc_init: clearing the workspace failed (%s)", hipGetErrorString(err));
  }
  err = hipStreamCreateWithFlags(&ctx->side, hipStreamNonBlocking);
  if (err == hipSuccess) err = hipEventCreateWithFlags(&ctx->fork, hipEventDisableTiming);
  if (err == hipSuccess) err = hipEventCreateWithFlags(&ctx->join, hipEventDisableTiming);
  if (err == hipSuccess) err = hipEventCreateWithFlags(&ctx->xfer, hipEventDisableTiming);
  if (err != hipSuccess) {
    if (ctx->side) (void)hipStreamDestroy(ctx->side);
    if (ctx->fork) (void)hipEventDestroy(ctx->fork);
    if (ctx->join) (void)hipEventDestroy(ctx->join);
    (void)hipFree(ctx->mem);
    delete ctx;
    return fail(GMC_ERR_HIP, "gmc_init: side stream or events (%s)", hipGetErrorString(err));
  }
  g_ctx = ctx;
  return GMC_OK;
}

int gmc_set_stream(void* stream) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ctx) return fail(GMC_ERR_STATE, "gmc_set_stream: no context");
  g_ctx->stream = static_cast<hipStream_t>(stream);
  return GMC_OK;
}

int64_t gmc_realized_k(int64_t N, int64_t K_req) {
  if (N < 1) return 0;
  return std::min<int64_t>(N, std::max<int64_t>(K_req, 1));
}

int64_t gmc_realized_budget(int64_t N, int64_t K_req, int64_t n_images) {
  if (N < 1 || n_images < 1) return 0;
  return std::min<int64_t>(N, std::max<int64_t>(K_req, n_images));
}

int gmc_compact_sequence(int64_t B, int64_t L, int64_t vis_start, int64_t N, int64_t K, const int32_t* out_idx,
                         int32_t* iota, int32_t* keep, const void* seq_rows, const void* vis_rows, void* out_rows,
                         int64_t row_bytes, const int32_t* seq_pos, int32_t* out_pos) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ctx) return fail(GMC_ERR_STATE, "gmc_compact_sequence: no context (call gmc_init first)");
  if (B < 1 || L < 1 || N < 1 || K < 1 || K > N || vis_start < 0 || vis_start + N > L || L > (1LL << 30))
    return fail(GMC_ERR_ARG, "gmc_compact_sequence: need B, L >= 1, 1 <= K <= N, 0 <= vis_start, vis_start + N <= L "
                "(B=%lld L=%lld vis_start=%lld N=%lld K=%lld)", static_cast<long long>(B), static_cast<long long>(L),
                static_cast<long long>(vis_start), static_cast<long long>(N), static_cast<long long>(K));
  if (!out_idx) return fail(GMC_ERR_ARG, "gmc_compact_sequence: out_idx is NULL");
  const int rows_set = (seq_rows != nullptr) + (vis_rows != nullptr) + (out_rows != nullptr);
  if (rows_set != 0 && rows_set != 3)
    return fail(GMC_ERR_ARG, "gmc_compact_sequence: seq_rows, vis_rows and out_rows must be all NULL or all set");
  if (rows_set == 3 && (row_bytes < 16 || row_bytes % 16 != 0 || row_bytes > (1LL << 24)))
    return fail(GMC_ERR_ARG, "gmc_compact_sequence: row_bytes=%lld must be a positive multiple of 16",
                static_cast<long long>(row_bytes));
  if ((seq_pos == nullptr) != (out_pos == nullptr))
    return fail(GMC_ERR_ARG, "gmc_compact_sequence: seq_pos and out_pos must be both NULL or both set");
  auto misaligned = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15u) != 0; };
  if (rows_set == 3 && (misaligned(seq_rows) || misaligned(vis_rows) || misaligned(out_rows)))
    return fail(GMC_ERR_ARG, "gmc_compact_sequence: rows must be 16-byte aligned");
  hipError_t err = hipSetDevice(g_ctx->device);
  if (err == hipSuccess)
    err = launch_compact_sequence(static_cast<int>(B), static_cast<int>(L), static_cast<int>(vis_start),
                                  static_cast<int>(N), static_cast<int>(K), out_idx, iota, keep, seq_rows, vis_rows,
                                  out_rows, rows_set == 3 ? static_cast<int>(row_bytes / 16) : 0, seq_pos, out_pos,
                                  g_ctx->stream);
  if (err != hipSuccess) return fail(GMC_ERR_HIP, "gmc_compact_sequence: %s", hipGetErrorString(err));
  return GMC_OK;
}

int gmc_gather_rows(int64_t n_tensors, const void* const* src, void* const* dst, int64_t n_seq,
                    int64_t seqs_per_keep, int64_t L, int64_t L2, int64_t row_bytes, const int32_t* keep) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ctx) return fail(GMC_ERR_STATE, "gmc_gather_rows: no context (call gmc_init first)");
  if (n_tensors < 1 || n_tensors > kMaxGather)
    return fail(GMC_ERR_ARG, "gmc_gather_rows: n_tensors=%lld out of [1, %d]", static_cast<long long>(n_tensors),
                kMaxGather);
  if (!src || !dst || !keep) return fail(GMC_ERR_ARG, "gmc_gather_rows: null pointer");
  if (n_seq < 1 || seqs_per_keep < 1 || n_seq % seqs_per_keep != 0 || L < 1 || L2 < 1 || L > (1LL << 30) ||
      L2 > (1LL << 30) || n_seq > 65535)
    return fail(GMC_ERR_ARG, "gmc_gather_rows: need n_seq in [1, 65535] a multiple of seqs_per_keep, L, L2 >= 1");
  if (row_bytes < 16 || row_bytes % 16 != 0 || row_bytes > (1LL << 24))
    return fail(GMC_ERR_ARG, "gmc_gather_rows: row_bytes=%lld must be a positive multiple of 16",
                static_cast<long long>(row_bytes));
  if (n_seq * L2 * (row_bytes / 16) >= (1LL << 31))
    return fail(GMC_ERR_ARG, "gmc_gather_rows: a destination tensor above 32 GiB; split the call");
  for (int64_t t = 0; t < n_tensors; ++t) {
    if (!src[t] || !dst[t]) return fail(GMC_ERR_ARG, "gmc_gather_rows: tensor %lld is NULL", static_cast<long long>(t));
    if ((reinterpret_cast<uintptr_t>(src[t]) | reinterpret_cast<uintptr_t>(dst[t])) & 15u)
      return fail(GMC_ERR_ARG, "gmc_gather_rows: tensor %lld is not 16-byte aligned", static_cast<long long>(t));
  }
  hipError_t err = hipSetDevice(g_ctx->device);
  if (err == hipSuccess)
    err = launch_gather_rows(static_cast<int>(n_tensors), src, dst, static_cast<int>(n_seq),
                             static_cast<int>(seqs_per_keep), static_cast<int>(L), static_cast<int>(L2),
                             static_cast<int>(row_bytes / 16), keep, g_ctx->stream);
  if (err != hipSuccess) return fail(GMC_ERR_HIP, "gmc_gather_rows: %s", hipGetErrorString(err));
  return GMC_OK;
}

int64_t gmc_workspace_bytes(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  return g_ctx ? static_cast<int64_t>(g_ctx->bytes) : 0;
}

const char* gmc_last_error(void) { return g_err; }

int gmc_timing_enable(int enable) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ctx) return fail(GMC_ERR_STATE, "gmc_timing_enable: no context");
  g_timer.on = enable != 0;
  return GMC_OK;
}

int gmc_timing_read(double* total_ms, int64_t* spans, int32_t n) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ctx) return fail(GMC_ERR_STATE, "gmc_timing_read: no context");
  if (!total_ms || !spans || n < kNumStages) return fail(GMC_ERR_ARG, "gmc_timing_read: need %d slots", kNumStages);
  for (int i = 0; i < n; ++i) { total_ms[i] = 0.0; spans[i] = 0; }
  hipError_t err = hipStreamSynchronize(g_ctx->stream);
  if (err != hipSuccess) return fail(GMC_ERR_HIP, "gmc_timing_read: %s", hipGetErrorString(err));
  for (const Span& sp : g_timer.spans) {
    float ms = 0.f;
    err = hipEventElapsedTime(&ms, sp.a, sp.b);
    if (err != hipSuccess) return fail(GMC_ERR_HIP, "hipEventElapsedTime: %s", hipGetErrorString(err));
    total_ms[sp.stage] += ms;
    spans[sp.stage] += 1;
  }
  g_timer.spans.clear();
  g_timer.used = 0;
  for (int i = 0; i < kNumStages; ++i) g_timer.open[i] = nullptr;
  return GMC_OK;
}

}  // extern "C"

namespace {

int make_shape(const Context& c, int64_t B, int64_t N, int64_t T, int64_t K_req, Shape* out, int64_t n_hist = 0,
               int64_t n_images = 1) {
  return gmc::resolve_shape(c.cfg, Limits{c.cap.B, c.cap.N, c.cap.T, c.cap.K, c.cfg.max_hist_views, c.cap.I}, B, N,
                            T, K_req, out, n_hist, n_images);
}

}  // namespace

namespace gmc {

int resolve_shape(const gmc_config& g, const Limits& cap, int64_t B, int64_t N, int64_t T, int64_t K_req,
                  Shape* out, int64_t n_hist, int64_t n_images) {
  if (B < 1) return fail(GMC_ERR_ARG, "batch=%lld must be >= 1", static_cast<long long>(B));
  if (N < 1) return fail(GMC_ERR_ARG, "N=%lld must be >= 1", static_cast<long long>(N));
  if (T < 0) return fail(GMC_ERR_ARG, "T=%lld must be >= 0", static_cast<long long>(T));
  if (B > cap.B) return fail(GMC_ERR_CAPACITY, "batch=%lld exceeds max_batch=%d", static_cast<long long>(B), cap.B);
  if (N > cap.N) return fail(GMC_ERR_CAPACITY, "N=%lld exceeds max_n=%d", static_cast<long long>(N), cap.N);
  if (T > cap.T) return fail(GMC_ERR_CAPACITY, "T=%lld exceeds max_t=%d", static_cast<long long>(T), cap.T);
  if (n_hist < 0) return fail(GMC_ERR_ARG, "n_hist=%lld must be >= 0", static_cast<long long>(n_hist));
  if (n_hist > cap.H)
    return fail(GMC_ERR_CAPACITY, "n_hist=%lld exceeds max_hist_views=%d", static_cast<long long>(n_hist), cap.H);
  if (n_images < 1) return fail(GMC_ERR_ARG, "n_images=%lld must be >= 1", static_cast<long long>(n_images));
  if (n_images > cap.I)
    return fail(GMC_ERR_CAPACITY, "n_images=%lld exceeds max_images=%d", static_cast<long long>(n_images), cap.I);
  if (n_images > N) return fail(GMC_ERR_ARG, "n_images=%lld exceeds N=%lld", static_cast<long long>(n_images),
                                static_cast<long long>(N));
  if (n_images > 1 && N > g.bounded_threshold_n)
    return fail(GMC_ERR_ARG, "multi-image prompts use the exact appearance bank: N=%lld exceeds %d",
                static_cast<long long>(N), g.bounded_threshold_n);
  const int64_t K = gmc_realized_budget(N, K_req, n_images);
  Shape s{};
  s.B = static_cast<int>(B);
  s.N = static_cast<int>(N);
  s.T = static_cast<int>(T);
  s.K = static_cast<int>(K);
  s.d = g.d;
  s.hq = g.n_q_heads;
  s.hkv = g.n_kv_heads;
  s.hg = g.n_q_heads / g.n_kv_heads;
  s.dh = g.head_dim;
  s.r = g.probe_rank;
  s.hr = s.hq * s.r;
  s.dtype = g.dtype;
  s.landmarks = g.landmarks;
  if (K < N && K > cap.K)
    return fail(GMC_ERR_CAPACITY, "realised K=%lld exceeds max_k=%d", static_cast<long long>(K), cap.K);
  s.bounded = N > g.bounded_threshold_n ? 1 : 0;
  s.app_rank = s.bounded ? g.app_rank : 0;
  // every message view contributes Hq T grounded rows (none without queries)
  s.nviews = s.T > 0 ? 1 + static_cast<int>(n_hist) : 1;
  s.mg1 = s.hq * s.T;
  s.mg = s.nviews * s.mg1;
  s.mv = app_rows(g, s.N);
  s.nimg = static_cast<int>(n_images);
  s.nseed = s.nimg > 1 ? s.nimg : 0;
  s.ms = g.landmarks * g.landmarks * s.nimg;
  s.m = s.mg + s.mv + s.ms;
  s.ldM = static_cast<int>(round_up(s.m, 4));
  s.b = s.bounded ? g.batch_b_bounded : g.batch_b;
  s.pool_cap = g.pool_mult * s.b;
  s.rounds = (K < N) ? static_cast<int>(cdiv(K - s.nseed, s.b)) : 0;
  s.ldK = static_cast<int>(round_up(K, 4));
  // column blocks of the appearance row statistics: 64-token tiles of the
  // exact Gram, smaller tiles of the bounded bank's GEMM
  s.n_app_cblk = static_cast<int>(cdiv(N, s.bounded ? kAppBoundedTile : 64));
  s.n_head_blk = static_cast<int>(cdiv(N, kHeadTok));
  {
    // split the logit columns until about two blocks per CU of a 256-CU part
    // are busy, keeping at least eight tiles (one per wave) per range
    const long long blocks = cdiv(static_cast<long long>(s.hg) * s.T, 16) * s.hkv * s.B;
    const long long ntile = cdiv(N, 16);
    long long ls = blocks > 0 ? 512 / blocks : 1;
    ls = std::min<long long>(ls, ntile / 8);
    s.lsplit = static_cast<int>(std::max<long long>(1, std::min<long long>(ls, kLogitSplit)));
  }
  s.npairs = s.hq * (s.hq + 1) / 2;
  *out = s;
  return GMC_OK;
}

int check_tensors(const Shape& s, const void* hidden, const void* text_q, const void* vis_k, const int32_t* pos3d,
                  const void* out_hidden, const int32_t* out_pos, const int32_t* out_idx, const gmc_view* hist) {
  if (!hidden || !vis_k || !pos3d || !out_hidden || !out_pos || !out_idx)
    return fail(GMC_ERR_ARG, "gmc_prune: null tensor pointer");
  if (s.T > 0 && !text_q) return fail(GMC_ERR_ARG, "gmc_prune: text_q is NULL with T > 0");
  if (s.nviews > 1) {
    if (!hist) return fail(GMC_ERR_ARG, "gmc_prune_views: hist is NULL with n_hist > 0");
    for (int v = 0; v + 1 < s.nviews; ++v)
      if (!hist[v].hidden || !hist[v].text_q || !hist[v].vis_k)
        return fail(GMC_ERR_ARG, "gmc_prune_views: historical view %d has a NULL tensor", v);
  }
  const size_t esz = s.dtype == GMC_F32 ? 4 : 2;
  // outputs must not overlap the inputs
  auto overlap = [](const void* a, size_t na, const void* b, size_t nb) {
    const char* x = static_cast<const char*>(a);
    const char* y = static_cast<const char*>(b);
    return x < y + nb && y < x + na;
  };
  const size_t n_hidden = esz * s.B * s.N * s.d, n_out = esz * s.B * s.K * s.d;
  const size_t n_pos = 12ull * s.B * s.N, n_opos = 12ull * s.B * s.K, n_idx = 4ull * s.B * s.K;
  const size_t n_q = esz * s.B * s.T * s.hq * s.dh, n_k = esz * s.B * s.N * s.hkv * s.dh;
  const void* ins[4] = {hidden, text_q, vis_k, pos3d};
  const size_t nins[4] = {n_hidden, text_q ? n_q : 0, n_k, n_pos};
  const void* outs[3] = {out_hidden, out_pos, out_idx};
  const size_t nouts[3] = {n_out, n_opos, n_idx};
  for (int o = 0; o < 3; ++o) {
    for (int i = 0; i < 4; ++i)
      if (nins[i] && overlap(outs[o], nouts[o], ins[i], nins[i]))
        return fail(GMC_ERR_ARG, "gmc_prune: output %d overlaps input %d", o, i);
    for (int o2 = o + 1; o2 < 3; ++o2)
      if (overlap(outs[o], nouts[o], outs[o2], nouts[o2]))
        return fail(GMC_ERR_ARG, "gmc_prune: outputs %d and %d overlap", o, o2);
  }
  return GMC_OK;
}

int enqueue_prune(const gmc_config& cfg, const Params& pr0, const Ws& ws, const Shape& s, const PathStreams& ps,
                  int diag, const void* hidden, const void* text_q, const void* vis_k, const int32_t* pos3d,
                  void* out_hidden, int32_t* out_pos, int32_t* out_idx, const float* nonvis_lse,
                  const gmc_trace& tr, bool* cert_done, const gmc_view* hist, const int32_t* image_id) {
  *cert_done = false;
  hipStream_t st = ps.st;
  hipError_t err;
  // message views: the current one, then the historical ones with their own
  // probes; the message mass beta_msg splits over them (reading R14)
  Params pr = pr0;
  MsgView views[kMaxViews] = {};
  views[0] = MsgView{hidden, text_q, vis_k, cfg.value_probe, cfg.value_probe_bias, nonvis_lse};
  const int n_hist = s.nviews - 1;
  if (n_hist > 0) {
    const size_t esz = s.dtype == GMC_F32 ? 4 : 2;
    pr.beta_view[0] = cfg.beta_msg * (1.f - cfg.hist_mass);
    for (int v = 1; v <= n_hist; ++v) {
      pr.beta_view[v] = cfg.beta_msg * cfg.hist_mass / static_cast<float>(n_hist);
      const char* probe = static_cast<const char*>(cfg.value_probe_hist) +
                          static_cast<size_t>(v - 1) * s.hq * s.r * s.d * esz;
      const float* bias = cfg.value_probe_bias_hist ? cfg.value_probe_bias_hist + (v - 1) * s.hq * s.r : nullptr;
      views[v] = MsgView{hist[v - 1].hidden, hist[v - 1].text_q, hist[v - 1].vis_k, probe, bias,
                         hist[v - 1].nonvis_lse};
    }
  }
  if (s.K == s.N) {
    err = launch_identity(s, hidden, pos3d, out_hidden, out_pos, out_idx, st);
    if (err != hipSuccess) return fail(GMC_ERR_HIP, "identity copy: %s", hipGetErrorString(err));
    return GMC_OK;
  }
  // a multi-image call first copies the (clamped) image ids and counts each
  // image's tokens; every later kernel, the bank stream's included, runs
  // after it
  if (s.nimg > 1) {
    err = launch_image_prep(s, ws, image_id, st);
    if (err != hipSuccess) return fail(GMC_ERR_HIP, "image ids: %s", hipGetErrorString(err));
  }
  // per-call reset and row norms (one kernel), then the bank kernels on the
  // side stream while the message kernels run on the caller's stream (they
  // write disjoint client rows).  Without a side stream (stage timing, the
  // static-scratch entry point) everything stays on one stream.
  const bool fork = ps.side != nullptr;
  // one image: the fork is a one-block gate on the side stream that waits for
  // this call's row-norm blocks (no event record on the caller's stream, whose
  // next kernel would wait for the command processor to process it).  The
  // gate of the next call may already wait while this call's selection runs,
  // so with several images, whose persistent selection takes every CU, an
  // event is used instead.
  const bool gate = fork && ps.call_tag != 0;
  err = launch_rownorm(s, ws, hidden, gate ? ps.call_tag : 0, st);
  if (err != hipSuccess) return fail(GMC_ERR_HIP, "row norms: %s", hipGetErrorString(err));
  hipStream_t bank_st = fork ? ps.side : st;
  if (gate) {
    err = launch_bank_gate(s, ws, ps.call_tag, ps.side);
    if (err != hipSuccess) return fail(GMC_ERR_HIP, "stream fork: %s", hipGetErrorString(err));
  } else if (fork) {
    err = hipEventRecord(ps.fork, st);
    if (err == hipSuccess) err = hipStreamWaitEvent(ps.side, ps.fork, 0);
    if (err != hipSuccess) return fail(GMC_ERR_HIP, "stream fork: %s", hipGetErrorString(err));
  }
  err = launch_banks(s, pr, ws, hidden, cfg.app_projection, pos3d, bank_st);
  if (err != hipSuccess) return fail(GMC_ERR_HIP, "bank kernels: %s", hipGetErrorString(err));
  // join: with text queries the last message kernel (one block per problem)
  // waits on a device flag that the side stream raises after its last bank
  // kernel, which costs less than an event wait on the caller's stream;
  // without text queries, an event
  int* bank_flag = ws.cnt + kCntBankFlag;   // cleared by the row-norm kernel
  const bool flag_join = fork && s.T > 0;
  if (flag_join) {
    err = launch_bank_signal(bank_flag, ps.side);
    if (err != hipSuccess) return fail(GMC_ERR_HIP, "stream join: %s", hipGetErrorString(err));
  } else if (fork) {
    err = hipEventRecord(ps.join, ps.side);
    if (err != hipSuccess) return fail(GMC_ERR_HIP, "stream join: %s", hipGetErrorString(err));
  }
  err = launch_message(s, pr, ws, views, tr.omega, flag_join ? bank_flag : nullptr, st);
  if (err != hipSuccess) return fail(GMC_ERR_HIP, "message kernels: %s", hipGetErrorString(err));
  if (fork && !flag_join) {
    err = hipStreamWaitEvent(st, ps.join, 0);
    if (err != hipSuccess) return fail(GMC_ERR_HIP, "stream join: %s", hipGetErrorString(err));
  }
  // per-round outputs of the selection: the trace's buffers, completed with
  // the workspace's certificate buffers when the certificate is computed
  const bool want_cert = (diag & GMC_DIAG_CERT) != 0 || (tr.round_gains && tr.round_scores);
  SelOut so{tr.round_pool, tr.round_batch, tr.round_gains, tr.round_scores};
  const bool cert = want_cert && s.rounds >= 1 && s.rounds <= ws.cert_rounds;
  if (cert) {
    if (!so.pool) so.pool = ws.cpool;
    if (!so.batch) so.batch = ws.cbat;
    if (!so.gains) so.gains = ws.cgain;
    if (!so.scores) so.scores = ws.cscore;
  }
  if (s.nimg > 1) {
    // S_0: the largest singleton gain of every image (after the banks joined)
    err = launch_image_seeds(s, ws, st);
    if (err != hipSuccess) return fail(GMC_ERR_HIP, "image seeds: %s", hipGetErrorString(err));
  }
  bool support_ready = false;
  err = launch_selection(s, pr, ws, so, st, &support_ready);
  if (err != hipSuccess) return fail(GMC_ERR_HIP, "selection kernels: %s", hipGetErrorString(err));
  err = launch_assignment(s, pr, ws, hidden, support_ready, tr.assign, st);
  if (err != hipSuccess) return fail(GMC_ERR_HIP, "assignment kernels: %s", hipGetErrorString(err));
  err = launch_transport(s, pr, ws, hidden, pos3d, out_hidden, out_pos, out_idx, st);
  if (err != hipSuccess) return fail(GMC_ERR_HIP, "transport kernels: %s", hipGetErrorString(err));
  if (cert) {
    err = launch_certificate(s, ws, so, st);
    if (err != hipSuccess) return fail(GMC_ERR_HIP, "certificate kernels: %s", hipGetErrorString(err));
    *cert_done = true;
  }
  if (diag & GMC_DIAG_FINITE) {
    err = launch_finite_scan(s, ws, out_hidden, st);
    if (err != hipSuccess) return fail(GMC_ERR_HIP, "non-finite scan: %s", hipGetErrorString(err));
  }
  if (tr.client || tr.stats || tr.ebar) {
    err = launch_trace_exports(s, ws, tr.client, tr.stats, tr.ebar, st);
    if (err != hipSuccess) return fail(GMC_ERR_HIP, "trace exports: %s", hipGetErrorString(err));
  }
  return GMC_OK;
}

}  // namespace gmc

namespace {

int run(int64_t B, const void* hidden, const void* text_q, const void* vis_k, const int32_t* pos3d,
        int64_t N, int64_t T, int64_t K, void* out_hidden, int32_t* out_pos, int32_t* out_idx,
        const float* nonvis_lse, const gmc_trace* trace, int64_t n_hist = 0, const gmc_view* hist = nullptr,
        const int32_t* image_id = nullptr, int64_t n_images = 1) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ctx) return fail(GMC_ERR_STATE, "gmc_prune: no context (call gmc_init first)");
  Context& c = *g_ctx;
  if (!image_id) n_images = 1;
  Shape s;
  int rc = make_shape(c, B, N, T, K, &s, n_hist, n_images);
  if (rc != GMC_OK) return rc;
  rc = check_tensors(s, hidden, text_q, vis_k, pos3d, out_hidden, out_pos, out_idx, hist);
  if (rc != GMC_OK) return rc;
  const gmc_trace tr = trace ? *trace : gmc_trace{};
  hipError_t err = hipSetDevice(c.device);
  if (err != hipSuccess) return fail(GMC_ERR_HIP, "hipSetDevice: %s", hipGetErrorString(err));
  hipStream_t st = c.stream;
  // the workspace is shared by every call: a call on another stream than the
  // previous one first waits for that stream (its selection may still read
  // the client matrix that this call's bank kernels rewrite)
  if (c.order_stream && st != c.order_stream) {
    err = hipEventRecord(c.xfer, c.order_stream);
    if (err == hipSuccess) err = hipStreamWaitEvent(st, c.xfer, 0);
    if (err != hipSuccess) return fail(GMC_ERR_HIP, "ordering after the previous call's stream: %s",
                                       hipGetErrorString(err));
  }
  c.has_call = true;
  c.last_stream = st;
  c.order_stream = st;
  c.last = s;
  c.last_identity = s.K == s.N;
  c.last_cert = false;
  // stage timing keeps every kernel on the caller's stream, so each stage's
  // span measures that stage alone
  PathStreams ps{st, g_timer.on ? nullptr : c.side, 0, c.fork, c.join};
  if (ps.side && s.B == 1 && s.K < s.N) {
    c.call_tag = c.call_tag == 0x7fffffff ? 1 : c.call_tag + 1;
    ps.call_tag = c.call_tag;
  }
  bool cert = false;
  rc = enqueue_prune(c.cfg, c.pr, c.ws, s, ps, c.diag, hidden, text_q, vis_k, pos3d, out_hidden, out_pos, out_idx,
                     nonvis_lse, tr, &cert, hist, image_id);
  c.last_cert = cert;
  return rc;
}

}  // namespace

extern "C" {

int gmc_prune(const void* hidden, const void* text_q, const void* vis_k, const int32_t* pos3d, int64_t N,
              int64_t T, int64_t K, void* out_hidden, int32_t* out_pos, int32_t* out_idx) {
  int64_t B;
  {
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_ctx) return fail(GMC_ERR_STATE, "gmc_prune: no context (call gmc_init first)");
    B = g_ctx->cfg.max_batch;
  }
  return run(B, hidden, text_q, vis_k, pos3d, N, T, K, out_hidden, out_pos, out_idx, nullptr, nullptr);
}

int gmc_prune_ex(int64_t B, const void* hidden, const void* text_q, const void* vis_k, const int32_t* pos3d,
                 int64_t N, int64_t T, int64_t K, void* out_hidden, int32_t* out_pos, int32_t* out_idx,
                 const float* nonvis_lse, const gmc_trace* trace) {
  return run(B, hidden, text_q, vis_k, pos3d, N, T, K, out_hidden, out_pos, out_idx, nonvis_lse, trace);
}

int gmc_prune_views(int64_t B, const void* hidden, const void* text_q, const void* vis_k, const int32_t* pos3d,
                    int64_t N, int64_t T, int64_t K, void* out_hidden, int32_t* out_pos, int32_t* out_idx,
                    const float* nonvis_lse, int64_t n_hist, const gmc_view* hist, const gmc_trace* trace) {
  return run(B, hidden, text_q, vis_k, pos3d, N, T, K, out_hidden, out_pos, out_idx, nonvis_lse, trace, n_hist,
             hist);
}

int gmc_prune_full(int64_t B, const void* hidden, const void* text_q, const void* vis_k, const int32_t* pos3d,
                   const int32_t* image_id, int64_t n_images, int64_t N, int64_t T, int64_t K, void* out_hidden,
                   int32_t* out_pos, int32_t* out_idx, const float* nonvis_lse, int64_t n_hist,
                   const gmc_view* hist, const gmc_trace* trace) {
  return run(B, hidden, text_q, vis_k, pos3d, N, T, K, out_hidden, out_pos, out_idx, nonvis_lse, trace, n_hist,
             hist, image_id, n_images);
}

int gmc_audit_message(int64_t B, int64_t N, int64_t T, int64_t K, const void* text_q, const void* vis_k,
                      const void* vis_v, const void* comp_k, const void* comp_v, const int32_t* carrier,
                      const float* weights, const float* nonvis_lse, float* rows_out, float* vec_out, float* out) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ctx) return fail(GMC_ERR_STATE, "gmc_audit_message: no context");
  Context& c = *g_ctx;
  if (B < 1 || N < 1 || T < 1 || K < 1 || K > N || N > kMaxN || T > (1 << 20))
    return fail(GMC_ERR_ARG, "gmc_audit_message: need B, T >= 1 and 1 <= K <= N <= %d", kMaxN);
  if (!text_q || !vis_k || !vis_v || !comp_k || !comp_v || !carrier || !out)
    return fail(GMC_ERR_ARG, "gmc_audit_message: null pointer");
  const gmc_config& g = c.cfg;
  Shape s{};
  s.B = static_cast<int>(B);
  s.N = static_cast<int>(N);
  s.T = static_cast<int>(T);
  s.K = static_cast<int>(K);
  s.d = g.d;
  s.hq = g.n_q_heads;
  s.hkv = g.n_kv_heads;
  s.hg = g.n_q_heads / g.n_kv_heads;
  s.dh = g.head_dim;
  s.dtype = g.dtype;
  s.mg1 = s.hq * s.T;
  // scratch inside the client-matrix buffer
  const long long mg1 = s.mg1;
  long long off = 0;
  auto take = [&](long long elems) { const long long o = off; off += (elems + 63) / 64 * 64; return o; };
  const long long oA = take(B * N * mg1), oY = take(B * mg1 * s.dh), oL = take(B * mg1), oM = take(B * K * mg1);
  const long long oO = take(B * (K + 1)), oMem = take(B * N), oC = take(B * K), oR = take(B * mg1 * kAuditRow);
  const long long cap = c.ws.s_E * c.cap.B;
  if (off > cap)
    return fail(GMC_ERR_CAPACITY, "gmc_audit_message: needs %lld floats of scratch, the client-matrix buffer holds %lld",
                off, cap);
  float* base = c.ws.E;
  AudWs aw{base + oA, base + oY, base + oL, base + oM, reinterpret_cast<int*>(base + oO),
           reinterpret_cast<int*>(base + oMem), reinterpret_cast<int*>(base + oC), base + oR};
  hipError_t err = hipSetDevice(c.device);
  hipStream_t st = c.stream;
  if (err == hipSuccess && c.order_stream && st != c.order_stream) {
    err = hipEventRecord(c.xfer, c.order_stream);
    if (err == hipSuccess) err = hipStreamWaitEvent(st, c.xfer, 0);
  }
  if (err == hipSuccess)
    err = launch_audit(s, aw, text_q, vis_k, vis_v, comp_k, comp_v, carrier, weights, nonvis_lse, rows_out, vec_out,
                       out, st);
  if (err != hipSuccess) return fail(GMC_ERR_HIP, "gmc_audit_message: %s", hipGetErrorString(err));
  c.order_stream = st;
  return GMC_OK;
}

int gmc_trace_dims_full(int64_t N, int64_t T, int64_t K, int64_t n_hist, int64_t n_images, int64_t* rounds,
                        int64_t* pool_cap, int64_t* batch_cap, int64_t* m_rows) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ctx) return fail(GMC_ERR_STATE, "gmc_trace_dims_full: no context");
  Shape s;
  const int rc = make_shape(*g_ctx, 1, N, T, K, &s, n_hist, n_images);
  if (rc != GMC_OK) return rc;
  if (rounds) *rounds = s.rounds;
  if (pool_cap) *pool_cap = s.pool_cap;
  if (batch_cap) *batch_cap = s.b;
  if (m_rows) *m_rows = s.m;
  return GMC_OK;
}

int gmc_set_diag(int32_t flags) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ctx) return fail(GMC_ERR_STATE, "gmc_set_diag: no context");
  if (flags & ~(GMC_DIAG_CERT | GMC_DIAG_FINITE)) return fail(GMC_ERR_ARG, "gmc_set_diag: unknown flags 0x%x", flags);
  g_ctx->diag = flags;
  return GMC_OK;
}

int gmc_get_diag(int64_t problem, gmc_diag* out) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ctx) return fail(GMC_ERR_STATE, "gmc_get_diag: no context");
  Context& c = *g_ctx;
  if (!c.has_call) return fail(GMC_ERR_STATE, "gmc_get_diag: no pruning call yet");
  if (!out) return fail(GMC_ERR_ARG, "gmc_get_diag: out is NULL");
  const Shape& s = c.last;
  if (problem < 0 || problem >= s.B)
    return fail(GMC_ERR_ARG, "gmc_get_diag: problem %lld outside [0, %d)", static_cast<long long>(problem), s.B);
  hipError_t err = hipSetDevice(c.device);
  if (err == hipSuccess) err = hipStreamSynchronize(c.last_stream);
  if (err == hipSuccess) err = hipStreamSynchronize(c.side);
  if (err != hipSuccess) return fail(GMC_ERR_HIP, "gmc_get_diag: %s", hipGetErrorString(err));
  const int p = static_cast<int>(problem);
  std::vector<int> cnt(static_cast<size_t>(c.cap.B) * kCounters);
  float st[kStats] = {};
  std::vector<float> cert;
  if (!c.last_identity) {
    err = launch_trace_exports(s, c.ws, nullptr, c.ws.dstat, nullptr, c.last_stream);
    if (err == hipSuccess) err = hipStreamSynchronize(c.last_stream);
    if (err == hipSuccess)
      err = hipMemcpy(st, c.ws.dstat + p * c.ws.s_dstat, sizeof(st), hipMemcpyDeviceToHost);
    if (err == hipSuccess && c.last_cert) {
      cert.resize(static_cast<size_t>(c.ws.s_cert));
      err = hipMemcpy(cert.data(), c.ws.cert + p * c.ws.s_cert, cert.size() * sizeof(float), hipMemcpyDeviceToHost);
    }
  }
  if (err == hipSuccess)
    err = hipMemcpy(cnt.data(), c.ws.cnt, cnt.size() * sizeof(int), hipMemcpyDeviceToHost);
  if (err == hipSuccess) err = launch_clear_status(c.ws, c.cap.B, c.last_stream);
  if (err == hipSuccess) err = hipStreamSynchronize(c.last_stream);
  if (err != hipSuccess) return fail(GMC_ERR_HIP, "gmc_get_diag: %s", hipGetErrorString(err));
  uint32_t status = 0;
  for (int q = 0; q < c.cap.B; ++q) status |= static_cast<uint32_t>(cnt[static_cast<size_t>(q) * kCounters + kCntStatus]);
  out->status = status;
  out->identity = c.last_identity ? 1 : 0;
  out->has_certificate = c.last_cert ? 1 : 0;
  out->k = s.K;
  out->rounds = c.last_identity ? 0 : s.rounds;
  out->m_rows = c.last_identity ? 0 : s.m;
  out->n_discarded = s.N - s.K;
  out->s_x = st[0];
  out->dbar = st[1];
  out->f_s = st[2];
  out->f_v = st[3];
  for (int b = 0; b < 3; ++b) {
    out->f_bank_s[b] = st[9 + b];
    out->f_bank_v[b] = st[12 + b];
  }
  out->c_b = 0.f;
  if (c.last_cert) {
    out->c_b = cert[static_cast<size_t>(c.ws.cert_rounds) * kCertFields];
    const int nr = std::min(s.rounds, std::max(out->max_rounds, 0));
    for (int r = 0; r < nr; ++r) {
      const float* ce = cert.data() + static_cast<size_t>(r) * kCertFields;
      if (out->u_top) out->u_top[r] = ce[0];
      if (out->gain) out->gain[r] = ce[1];
      if (out->q) out->q[r] = ce[2];
      if (out->pool_margin) out->pool_margin[r] = ce[3];
      if (out->batch_margin) out->batch_margin[r] = ce[4];
    }
  }
  if (status & (kStatusSelect | kStatusBank))
    return fail(GMC_ERR_DEVICE, "a bounded device wait timed out (status 0x%x): the results are invalid", status);
  if (status & kStatusNonfinite)
    return fail(GMC_ERR_NONFINITE, "a non-finite value was met (status 0x%x)", status);
  return GMC_OK;
}

int gmc_trace_dims(int64_t N, int64_t T, int64_t K, int64_t* rounds, int64_t* pool_cap, int64_t* batch_cap,
                   int64_t* m_rows) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ctx) return fail(GMC_ERR_STATE, "gmc_trace_dims: no context");
  Shape s;
  const int rc = make_shape(*g_ctx, 1, N, T, K, &s);
  if (rc != GMC_OK) return rc;
  if (rounds) *rounds = s.rounds;
  if (pool_cap) *pool_cap = s.pool_cap;
  if (batch_cap) *batch_cap = s.b;
  if (m_rows) *m_rows = s.m;
  return GMC_OK;
}

}  // extern "C"
