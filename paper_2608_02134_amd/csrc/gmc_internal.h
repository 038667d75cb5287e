// Shapes, settings and workspace layout shared by the host sequencer and the
// kernels of the GMC operator.  Plain structs, passed to kernels by value.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gmc {

constexpr int kMaxHeads = 32;     // Hq limit (head-pattern Gram kept in registers)
constexpr int kMaxViews = 4;      // message views: the current one + up to 3 historical
constexpr int kMaxProbe = 8;      // probe rank limit
constexpr int kMaxN = 32768;      // tokens per problem (top-k keys live in LDS)
constexpr int kHeadTok = 8;       // tokens per head-Gram block (two per wave)
constexpr int kStats = 15;
constexpr int kCounters = 8;      // completion counters per problem
constexpr int kCntBankFlag = 6;   // slot of problem 0: the bank kernels of the call have finished
constexpr int kCntStatus = 7;     // device status bits (sticky; cleared from the host only)
constexpr unsigned kStatusSelect = 1u;    // a hand-off wait of the persistent selection timed out
constexpr unsigned kStatusBank = 2u;      // the bank stream's gate or join timed out
constexpr unsigned kStatusNonfinite = 4u; // debug scan: a non-finite value
constexpr unsigned kStatusInput = 8u;     // image ids out of range / an image without tokens
constexpr int kMaxImages = 64;            // GMC_MAX_IMAGES
// Bounded waits of the bank stream, in ticks of the 100 MHz constant clock:
// the start gate may wait behind everything the caller queued before the
// call, so it gives up only after 10 s; the join waits for bank kernels that
// run concurrently, 2 s.
constexpr unsigned long long kGateWaitTicks = 1000000000ull;
constexpr unsigned long long kJoinWaitTicks = 200000000ull;
constexpr int kCertMaxRounds = 64;   // GMC_CERT_MAX_ROUNDS
constexpr int kAuditRow = 8;         // GMC_AUDIT_ROW: per-client audit statistics
constexpr int kAuditOut = 8;         // GMC_AUDIT_OUT: per-problem audit results
constexpr int kCertFields = 5;       // U_t, gain, q_t, pool margin, batch margin
constexpr int kMaxPersist = 256;  // blocks per problem of the persistent selection
constexpr int kMaxGather = 64;    // tensors per row-gather launch (GMC_MAX_GATHER_TENSORS)
constexpr int kLogitSplit = 16;   // column ranges of the message-logit kernels (at most)
constexpr int kProbeSplit = 4;    // K splits of the value-probe GEMM (d a multiple of 256)
constexpr int kAppBoundedTile = 32;   // tile of the bounded appearance GEMM (fp32 operands, rank-long)

// Call shape, resolved on the host for one gmc_prune call.
struct Shape {
  int B, N, T, K, d, hq, hkv, dh, r, hr;  // hr = hq * r
  int hg;                                 // query heads per kv head
  int mg, mv, ms, m;                      // client rows: grounded, appearance, spatial, total
  int nviews, mg1;                        // message views; grounded rows per view (mg = nviews mg1)
  int nimg, nseed;                        // images; seeds before the rounds (nimg when nimg > 1, else 0)
  int ldM;                                // token-major client matrix: floats per token (multiple of 4, >= m)
  int bounded;                            // 1: bounded appearance bank
  int app_rank;
  int b, pool_cap, rounds;                // selection batch, pool capacity, rounds
  int ldK;                                // cosine buffer row stride (floats)
  int n_app_cblk;                         // column blocks of the appearance GEMM
  int n_head_blk;                         // token blocks of the head-Gram kernel
  int lsplit;                             // column ranges of the message-logit kernels
  int npairs;                             // head pairs h <= g
  int landmarks;
  int dtype;                              // 0 float32, 1 bfloat16
};

// Frozen settings (copied from gmc_config).
struct Params {
  float lambda_mass, eps_mass, beta_msg, beta_app, beta_spa, tau_v, tau_s;
  float tau_r, resp_eps, spatial_w, gate_t, gate_p, amb_margin, amb_p;
  int g_form;
  float pop_strength, tau_j;
  int max_head_clusters;
  float disp_eps, terminal_q_weight, rms_eps, norm_eps, restore_eps;
  int pool_mult;
  const float* probe_bias;   // [hq][r] or null: b_h added to Z_h[i] (of the view being built)
  float beta_view[kMaxViews];   // mass of each message view (current first)
};

// Workspace: every buffer is [max_batch][per-problem size]; s_* are the
// per-problem strides in elements.
struct Ws {
  float* n2;       long long s_n;       // squared row norms            [N]
  float* z;        long long s_z;       // probe coordinates Z          [N][hr]
  float* zp;       long long s_zp;      // split-K probe partials       [kProbeSplit][N][hr]
  float* lpart;    long long s_lpart;   // message-logit range partials  [4][kLogitSplit][mg]
  int* lcnt;       long long s_lcnt;    // range arrivals per logit row tile [ceil(hg T/16) hkv]
  float* sig;      long long s_sig;     // mass coordinate sigma_h      [hq]
  float* ell;      long long s_ell;     // ||Z_h[i]||^2; the atom norm is sqrt(ell + sigma_h^2)  [hq][N]
  float* E;        long long s_E;       // client energies, token-major [N][ldM]
  float* alpha;    long long s_m;       // row pre-weights              [ldM]
  float* peak;                          // max_i Cbar_mi                [ldM]
  float* rowsum;                        // grounded row sums Z_(h,t)    [ldM]
  float* apart_sum; float* apart_max; long long s_apart;  // appearance partials [cblk][mv]
  float* gpart;    long long s_gpart;   // head-Gram partials, per view [views][blk][npairs]
  long long s_gpart1;                   // one view's share of gpart
  float* n2h;      long long s_n2h;     // squared row norms of a historical view's states [N]
  int* img;        long long s_img;     // image of every token (clamped ids)  [N]
  int* imgcnt;     long long s_imgcnt;  // tokens per image                    [kMaxImages]
  float* e2;       long long s_e2;      // sum_t nu_t e^2               [hq][N]
  float* omega;    long long s_om;      // head weights                 [kMaxHeads]
  float* ebar;     long long s_eb;      // normalised energy            [N]
  float* pc;       long long s_pc;      // spatial coordinates          [N][2]
  float* bounds;   long long s_bd;      // grid origin/extent           [4]
  float* y;        long long s_y;       // projected states (bounded)   [N][app_rank]
  int* clients;    long long s_cl;      // bounded appearance clients   [mv]
  float* cov;      long long s_cov;     // coverage maxima b_m          [ldM]
  int* sel;        long long s_sel;     // round that selected i, -1    [N]
  int* order;      long long s_ord;     // support in selection order   [N]
  int* pool;       long long s_pool;    // current pool                 [pool_cap]
  float* spart;    long long s_spart;   // score partials per row chunk [2][ceil(M/64)][64]
  int* batch;      long long s_bat;     // last batch                   [b]
  int* slot;       long long s_slot;    // rank of a selected token     [N]
  int* sup;        long long s_sup;     // support, ascending           [N]
  float* cosb;     long long s_cos;     // cos to support               [N][ldK]
  float* delta;    long long s_del;     // selected-cosine gap          [N]
  float* gate;     long long s_gate;    // s_x, mean gap                [4]
  int* ftag;       long long s_ftag;    // row-norm blocks done: call number [ceil(N/4)]
  int* pi;         long long s_pi;      // assignment                   [N]
  float* stats;    long long s_st;      // diagnostics                  [kStats]
  uint32_t* keys;  long long s_keys;    // top-k keys when N exceeds LDS [N]
  float* u;        long long s_u;       // reduced singleton gains      [N]
  int* cnt;        long long s_cnt;     // completion counters          [kCounters]
  float* rstat;    long long s_rstat;   // large-pool row statistics    [3][ldM]
  float* lstat;    long long s_lstat;   // landmark min distance        [L*L]
  // persistent selection: values tagged with (round + 1) in the high word,
  // double-buffered by round parity; zeroed at the start of every call
  unsigned long long* tu; long long s_tu;  // tagged gains               [2][N]
  unsigned long long* ts; long long s_ts;  // tagged score partials [2][ceil(M/64)][64], then the pool [2][64]
  unsigned long long* tc; long long s_tc;  // tagged coverage + heartbeats [2][ldM + kMaxPersist]
  // diagnostics (certificate of the selection rounds, exported statistics);
  // the per-round buffers are indexed flat as (p * rounds + r) * row, so a
  // call of at most cert_rounds rounds fits
  int cert_rounds;                      // round capacity of the buffers below
  float* cgain;    long long s_cgain;   // each round's gains           [cert_rounds][N]
  float* cscore;   long long s_cscore;  // each round's pool scores     [cert_rounds][pool_cap]
  int* cpool;      long long s_cpool;   // each round's pool            [cert_rounds][pool_cap]
  int* cbat;       long long s_cbat;    // each round's batch           [cert_rounds][bmax]
  float* cpart;    long long s_cpart;   // coverage-gain block partials [cert_rounds][ceil(ldM/256)]
  float* cert;     long long s_cert;    // per-round certificate        [cert_rounds][kCertFields] + c_B
  float* dstat;    long long s_dstat;   // exported statistics          [kStats]
};

// Per-round outputs of the selection kernels (all optional): pools and
// batches as the trace lays them out, the gains of every token and the pool
// scores; entry (p, r) starts at (p * rounds + r) times the row length.
struct SelOut {
  int32_t* pool;    // [pool_cap]
  int32_t* batch;   // [b]
  float* gains;     // [N]
  float* scores;    // [pool_cap]
};

#ifdef __HIPCC__
// Records device status bits of problem p's counters (sticky OR).
__device__ __forceinline__ void raise_status(int* cnt, unsigned bits) {
  __hip_atomic_fetch_or(reinterpret_cast<unsigned*>(&cnt[kCntStatus]), bits, __ATOMIC_RELAXED,
                        __HIP_MEMORY_SCOPE_AGENT);
}

// Per-call state of problem p, over a grid-stride range (x0, stride): nothing
// selected, coverage and row-weight padding zero, tagged hand-off buffers and
// completion counters cleared.  Runs inside the first kernel of a call.
__device__ __forceinline__ void call_init_range(const Shape& sh, const Ws& ws, int p, int x0, int stride) {
  for (int i = x0; i < sh.N; i += stride) {
    ws.sel[p * ws.s_sel + i] = -1;
    ws.tu[p * ws.s_tu + i] = 0ull;
    ws.tu[p * ws.s_tu + sh.N + i] = 0ull;
  }
  for (int m = x0; m < sh.ldM; m += stride) {
    ws.cov[p * ws.s_cov + m] = 0.f;
    if (m >= sh.m) ws.alpha[p * ws.s_m + m] = 0.f;
  }
  for (int j = x0; j < 128 * ((sh.m + 63) / 64) + 128; j += stride) ws.ts[p * ws.s_ts + j] = 0ull;
  for (int j = x0; j < 2 * (sh.ldM + kMaxPersist); j += stride) ws.tc[p * ws.s_tc + j] = 0ull;
  for (int j = x0; j < (sh.hg * sh.T + 15) / 16 * sh.hkv; j += stride) ws.lcnt[p * ws.s_lcnt + j] = 0;
  // written through: the bank stream raises its flag in these words; the
  // status word is sticky (the host clears it after reading it)
  if (x0 < kCounters && x0 != kCntStatus)
    __hip_atomic_store(&ws.cnt[p * ws.s_cnt + x0], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
#endif

}  // namespace gmc
