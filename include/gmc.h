/*
 * gmc.h - C-ABI of the MI355X (gfx950) GMC boundary operator library.
 *
 * GMC (Grounded Message Coreset pruning) compresses the N visual states of
 * a vision-language decoder at a boundary layer p to K carriers:
 *   1. native message clients from the text-query -> visual-key softmax
 *      slice (Sec. 3.2; App. H Eq. cond-native-message, Eq.
 *      cond-mass-coordinate, Eq. cond-grounded-client), with farthest-first
 *      head clusters (Eq. cond-head-pattern, Eq. cond-head-weight);
 *   2. appearance and spatial clients (Eq. cond-aux-clients) pre-weighted
 *      into one facility-location objective (Eq. coverage, Eq. cond-coverage);
 *   3. batched responsibility selection of K carriers (Eq. responsibility,
 *      Eq. cond-responsibility), budget K = min{N, max{K_r, 1}}
 *      (Sec. 3.1 problem formulation);
 *   4. population assignment (Eq. cond-assignment, Eq.
 *      cond-population-gate) and weighted-centroid transport with RMS
 *      restoration (Eq. transport, Eq. cond-transport, Eq.
 *      cond-grounded-energy);
 *   5. physical compaction keeping each carrier's original (t,h,w) position
 *      ids (App. H "Index map and physical token accounting").
 *
 * Conventions shared by every entry point:
 *   - Tensor pointers are DEVICE pointers owned by the caller, unless stated.
 *     The library keeps no reference to them after a call returns, except
 *     value_probe / app_projection in gmc_config, which must stay valid until
 *     gmc_free().
 *   - Work is enqueued asynchronously on the stream set by gmc_set_stream
 *     (default: the null stream).  Outputs are valid once that stream has
 *     synchronised.  Host-side validation happens before anything is enqueued.
 *   - Row-major layouts; "dtype" is the element type chosen in gmc_config
 *     (float32 or bfloat16 stored as its 16-bit pattern).
 *   - Return value 0 on success, a negative GMC_ERR_* code otherwise;
 *     gmc_last_error() then describes the failure.  A failed call enqueues
 *     nothing and leaves the outputs untouched.
 *   - One library context per process; calls are serialised by an internal
 *     mutex and share one workspace.  Consecutive pruning calls are ordered
 *     on the device even when gmc_set_stream changed the stream in between
 *     (the new stream first waits for the previous call's stream).
 */
#ifndef GMC_H
#define GMC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GMC_OK 0
#define GMC_ERR_ARG (-1)      /* null pointer, bad size, bad config value      */
#define GMC_ERR_CAPACITY (-2) /* call exceeds the capacities given at init     */
#define GMC_ERR_STATE (-3)    /* no context (gmc_init not called / failed)     */
#define GMC_ERR_HIP (-4)      /* HIP runtime failure (no device, launch, OOM)  */
#define GMC_ERR_DEVICE (-5)   /* gmc_get_diag: a bounded device wait of an
                                 earlier call timed out (its results are invalid) */
#define GMC_ERR_NONFINITE (-6) /* gmc_get_diag, debug mode: an earlier call met a
                                  non-finite value (App. J numerical checks)    */

/* Device status bits (sticky: set by the kernels of any call, cleared only by
 * gmc_get_diag, which reports and clears them).                              */
#define GMC_STATUS_SELECT_TIMEOUT 1u /* a hand-off wait of the persistent selection */
#define GMC_STATUS_BANK_TIMEOUT 2u   /* the bank stream's start gate or its join     */
#define GMC_STATUS_NONFINITE 4u      /* debug mode: a non-finite client energy, row
                                        weight or output value                      */
/* GMC_STATUS_INPUT (8): see gmc_prune_full                                           */

#define GMC_F32 0
#define GMC_BF16 1

/* Number of float entries gmc_trace.stats receives per problem. */
#define GMC_STATS 15
/* stats layout: [0] s_x  [1] mean selected-cosine gap over discarded tokens
 *               [2] F(S)  [3] F(V)  [4] realised K  [5] rounds  [6] M rows
 *               [7] number of discarded tokens
 *               [8] device status bits (GMC_STATUS_*), sticky until
 *                   gmc_get_diag clears them: nonzero means a bounded device
 *                   wait timed out or (debug mode) a non-finite value was met;
 *                   the results of that call are invalid
 *               [9..11]  F_b(S) of the grounded, appearance, spatial bank
 *               [12..14] F_b(V) of the same banks; omega_b = F_b(V)/F(V)
 *                   and c_b = F_b(S)/F_b(V) (Eq. cond-bank-mixture)       */

/*
 * gmc_config - model shape, capacities and the frozen settings.
 * gmc_config_default() fills the settings of the paper's configuration table
 * (App. H, Table cond-config) and the readings documented with the library;
 * the caller then sets the shape, capacity and pointer fields.
 */
typedef struct gmc_config {
  /* model shape */
  int32_t d;            /* hidden size, multiple of 64                          */
  int32_t n_q_heads;    /* Hq, 1..32                                             */
  int32_t n_kv_heads;   /* Hkv, divides Hq; query head h reads kv head h*Hkv/Hq   */
  int32_t head_dim;     /* dh, multiple of 32, <= 256                            */
  int32_t probe_rank;   /* r, 1..8 (paper: 4)                                    */
  int32_t dtype;        /* GMC_F32 or GMC_BF16 for hidden/text_q/vis_k/out      */
  /* capacities: the workspace is sized once, in gmc_init, for these         */
  int32_t max_batch;    /* problems per call (gmc_prune uses exactly this many) */
  int32_t max_n;        /* visual tokens per problem, <= 32768                  */
  int32_t max_t;        /* text queries per problem                             */
  int32_t max_k;        /* realised budget per problem (0: max_n)               */
  /* device inputs fixed for the context's lifetime (caller-owned)           */
  const void* value_probe;    /* [Hq][r][d] dtype: per-head folded value path
                                 G_h = (W^V_kv(h) O_h P)^T (Eq. cond-mass-
                                 coordinate); required                       */
  const void* app_projection; /* [app_rank][d] dtype, entries +-1: the fixed
                                 Rademacher map of the bounded appearance bank
                                 (App. H "Appearance and spatial clients");
                                 required iff max_n > bounded_threshold_n     */
  /* frozen settings (Table cond-config) */
  float lambda_mass, eps_mass;          /* 1, 1e-8                            */
  float beta_msg, beta_app, beta_spa;   /* 1, 0.5, 0.25                       */
  float tau_v, tau_s;                   /* 0.2, 0.02                          */
  int32_t landmarks;                    /* 16 (16 x 16 spatial clients)       */
  int32_t batch_b, pool_mult;           /* 16, 4                              */
  float tau_r, resp_eps;                /* 0.1, 1e-30                         */
  float spatial_w, gate_t, gate_p;      /* 0.5, 0.08, 8                       */
  float amb_margin, amb_p;              /* 0.05, 8                            */
  int32_t g_form;                       /* 0 smooth exp(-(d/m)^p), 1 hard     */
  float pop_strength, tau_j;            /* 0.5, 1                             */
  int32_t max_head_clusters;            /* 4                                  */
  float disp_eps, terminal_q_weight;    /* 0.05, 2                            */
  float rms_eps, norm_eps, restore_eps; /* 1e-6, 1e-12, 1e-6                  */
  int32_t bounded_threshold_n;          /* 4096: N above it uses the bounded bank */
  int32_t app_rank, app_max_clients;    /* 128, 4096                          */
  int32_t batch_b_bounded;              /* 512                                */
  /* optional device input fixed for the context's lifetime (caller-owned)  */
  const float* value_probe_bias; /* [Hq][r] fp32 or NULL (zero): the value
                                    projection's bias carried through the same
                                    folded path, b_h = b^V_kv(h) O_h P, for
                                    models whose V projection has a bias; then
                                    Z_h[i] = x~_i G_h + b_h (Eq. cond-mass-
                                    coordinate with V = x~ W^V + b^V)        */
  /* completed historical message views (App. H "Native message clients";
     Table cond-config: current/history mass 0.5/0.5, two views); used by
     gmc_prune_views                                                       */
  int32_t max_hist_views;       /* 0..GMC_MAX_HIST_VIEWS (default 0)        */
  float hist_mass;              /* share of beta_msg the historical views
                                   carry together, split equally (0.5); the
                                   current view carries the rest           */
  const void* value_probe_hist; /* [max_hist_views][Hq][r][d] dtype: each
                                   view's folded probe (W^V O_h P of that
                                   view's block); required iff
                                   max_hist_views > 0 (caller-owned, kept)  */
  const float* value_probe_bias_hist; /* [max_hist_views][Hq][r] fp32 or NULL */
  /* multi-image prompts (Sec. 3.1; App. H), used by gmc_prune_full          */
  int32_t max_images;           /* images per problem, 1..GMC_MAX_IMAGES (0 = 1) */
} gmc_config;

/*
 * gmc_trace - optional device buffers the operator fills for inspection
 * (tests, diagnostics).  Every pointer may be NULL.  Sizes come from
 * gmc_trace_dims().  Problem p's block starts at p times the per-problem
 * size.
 */
typedef struct gmc_trace {
  int32_t* round_pool;  /* [B][rounds][pool_cap]: each round's candidate pool,
                           ascending source index, -1 padded                  */
  int32_t* round_batch; /* [B][rounds][batch_cap]: each round's batch,
                           ascending source index, -1 padded                  */
  int32_t* assign;      /* [B][N]: representative pi(i) (source index)        */
  float* omega;         /* [B][Hq]: head weights omega_h                       */
  float* ebar;          /* [B][N]: normalised grounded energy ebar_i           */
  float* client;        /* [B][m_rows][N]: pre-weighted client matrix Cbar    */
  float* stats;         /* [B][GMC_STATS]: see GMC_STATS                       */
  float* round_gains;   /* [B][rounds][N]: each round's singleton gains
                           u_i = sum_m [Cbar_mi - b_m(S_t)]_+ as the selection
                           computed them (Eq. cond-responsibility), 0 for tokens
                           selected in earlier rounds                         */
  float* round_scores;  /* [B][rounds][pool_cap]: each round's responsibility
                           scores s_i of the pool, in round_pool's order
                           (ascending source index), 0 padded                 */
} gmc_trace;

/* Fill *cfg with the frozen settings; shape/capacity/pointers are zeroed. */
void gmc_config_default(gmc_config* cfg);

/*
 * gmc_init - validate *cfg, create the context and allocate its workspace
 * (one device allocation sized from the capacities).  Replaces any existing
 * context.  The config struct is copied; the two device pointers in it are
 * borrowed.  Errors: GMC_ERR_ARG (bad field), GMC_ERR_HIP (no device, OOM).
 */
int gmc_init(const gmc_config* cfg);

/* Use `stream` (a hipStream_t, or NULL for the null stream) for all
 * subsequent work.  Errors: GMC_ERR_STATE. */
int gmc_set_stream(void* stream);

/*
 * gmc_prune - run the operator on cfg.max_batch independent problems.
 *   hidden     [B][N][d]        dtype   visual residual states h_i at boundary p
 *   text_q     [B][T][Hq][dh]   dtype   text queries (post-norm, post-rotary)
 *   vis_k      [B][N][Hkv][dh]  dtype   visual keys (post-norm, post-rotary)
 *   pos3d      [B][N][3]        int32   original (t,h,w) multimodal position ids
 *   N >= 1, T >= 0 (T = 0: no grounded clients, uniform energy), K = requested
 *   budget K_r; the realised K = gmc_realized_k(N, K_r).
 *   out_hidden [B][K][d]  dtype  transported carriers, ascending source order
 *   out_pos    [B][K][3]  int32  the carriers' original position ids
 *   out_idx    [B][K]     int32  the carriers' source indices, ascending
 * K = N returns the inputs unchanged (identity).  Outputs must not overlap
 * inputs.  Errors: GMC_ERR_ARG, GMC_ERR_CAPACITY, GMC_ERR_STATE, GMC_ERR_HIP.
 */
int gmc_prune(const void* hidden, const void* text_q, const void* vis_k, const int32_t* pos3d,
              int64_t N, int64_t T, int64_t K, void* out_hidden, int32_t* out_pos,
              int32_t* out_idx);

/*
 * gmc_prune_ex - gmc_prune with an explicit problem count 1 <= B <= max_batch
 * and two optional extras:
 *   nonvis_lse [B][Hq][T] float32 or NULL: log-sum-exp of each query's logits
 *              over the preceding nonvisual keys, so the visual slice keeps the
 *              native softmax denominator (Eq. cond-native-message); NULL
 *              means visual keys only.
 *   trace      host struct of optional device buffers (see gmc_trace), or NULL.
 */
int gmc_prune_ex(int64_t B, const void* hidden, const void* text_q, const void* vis_k,
                 const int32_t* pos3d, int64_t N, int64_t T, int64_t K, void* out_hidden,
                 int32_t* out_pos, int32_t* out_idx, const float* nonvis_lse,
                 const gmc_trace* trace);

/*
 * Diagnostics (Prop. 1 Eq. deployed-approximation; App. I Eq. cond-final-cert,
 * Eq. cond-bank-mixture; App. J numerical checks).
 *
 * gmc_set_diag - flags for subsequent calls (0 by default):
 *   GMC_DIAG_CERT    log the deployed batched-solver certificate of every
 *                    selection round of the call: U_t = the sum of the K
 *                    largest remaining singleton gains, the round's coverage
 *                    gain F(S_t u B_t) - F(S_t), q_t = gain / U_t (0 when
 *                    U_t = 0), c_B = 1 - prod_t (1 - q_t), and the decision
 *                    margins (relative pool and batch cut gaps).  Computed on
 *                    the device from the selection's own gains and scores,
 *                    for calls of at most GMC_CERT_MAX_ROUNDS rounds (and the
 *                    context's round capacity); extra kernels, no effect on
 *                    the outputs.
 *   GMC_DIAG_FINITE  scan the client matrix, row weights and outputs of
 *                    every call for non-finite values (sets
 *                    GMC_STATUS_NONFINITE).
 * Errors: GMC_ERR_STATE, GMC_ERR_ARG (unknown flag).
 */
#define GMC_DIAG_CERT 1
#define GMC_DIAG_FINITE 2
#define GMC_CERT_MAX_ROUNDS 64
int gmc_set_diag(int32_t flags);

/*
 * gmc_diag - host-side diagnostics of the last pruning call (one problem).
 * The per-round arrays are caller-owned HOST arrays of max_rounds entries,
 * or NULL; entries past `rounds` are left untouched.
 */
typedef struct gmc_diag {
  uint32_t status;        /* OR of every problem's device status bits (GMC_STATUS_*) */
  int32_t identity;       /* 1: the last call returned its inputs (K = N)            */
  int32_t has_certificate;/* 1: the per-round certificate below was computed         */
  int32_t k, rounds, m_rows, n_discarded;
  float s_x, dbar;        /* separability gate, mean selected-cosine gap             */
  float f_s, f_v;         /* F(S), F(V)                                              */
  float f_bank_s[3], f_bank_v[3]; /* F_b(S), F_b(V): grounded, appearance, spatial   */
  float c_b;              /* 1 - prod_t (1 - q_t)  (Prop. 1)                         */
  int32_t max_rounds;     /* capacity of the arrays below                            */
  float* u_top;           /* [rounds] U_t                                            */
  float* gain;            /* [rounds] F(S_t u B_t) - F(S_t)                          */
  float* q;               /* [rounds] q_t                                            */
  float* pool_margin;     /* [rounds] (u_(p) - u_(p+1)) / u_(1), p = pool size;
                             INFINITY when the cut is between exact zeros or the
                             pool takes every remaining token                     */
  float* batch_margin;    /* [rounds] (s_(b) - s_(b+1)) / s_(1), b = batch size   */
} gmc_diag;

/*
 * gmc_get_diag - synchronise the context's streams, fill *out for problem
 * `problem` (0 <= problem < B) of the last gmc_prune / gmc_prune_ex call,
 * then clear the device status bits.  Returns GMC_ERR_DEVICE when a
 * timeout bit was set, GMC_ERR_NONFINITE when the non-finite bit was set
 * (out is filled in both cases), GMC_ERR_STATE without a context or a
 * call, GMC_ERR_ARG for a bad problem index or NULL out, GMC_ERR_HIP.
 */
int gmc_get_diag(int64_t problem, gmc_diag* out);

/*
 * gmc_prune_views - gmc_prune_ex with n_hist completed historical message
 * views (App. H "Native message clients"; Eq. cond-head-pattern; Table
 * cond-config).  Each view is a separate collection of grounded client rows
 * built exactly like the current view's, from the view's own states, queries,
 * keys and folded value probe (config.value_probe_hist[v]); its rows carry
 * mass hist_mass * beta_msg / n_hist and the current view's
 * (1 - hist_mass) * beta_msg.  Head weights come from the head patterns
 * concatenated over the views (each view's atoms scaled to unit average norm
 * and by sqrt of its mass); the population energy from the current view.
 *   hist[v].hidden     [B][N][d]        dtype  states entering the view's block
 *   hist[v].text_q     [B][T][Hq][dh]   dtype  the view's text queries (same T)
 *   hist[v].vis_k      [B][N][Hkv][dh]  dtype  the view's visual keys
 *   hist[v].nonvis_lse [B][Hq][T] fp32 or NULL
 * 0 <= n_hist <= config.max_hist_views; n_hist = 0 is gmc_prune_ex.  With
 * T = 0 there are no grounded rows and the views are not read.  The trace's
 * client matrix then holds the current view's grounded rows, then each
 * historical view's, then the appearance and spatial rows.  Errors: as
 * gmc_prune_ex, GMC_ERR_CAPACITY for n_hist above the capacity.
 */
#define GMC_MAX_HIST_VIEWS 3
typedef struct gmc_view {
  const void* hidden;
  const void* text_q;
  const void* vis_k;
  const float* nonvis_lse;
} gmc_view;
int gmc_prune_views(int64_t B, const void* hidden, const void* text_q, const void* vis_k, const int32_t* pos3d,
                    int64_t N, int64_t T, int64_t K, void* out_hidden, int32_t* out_pos, int32_t* out_idx,
                    const float* nonvis_lse, int64_t n_hist, const gmc_view* hist, const gmc_trace* trace);

/*
 * gmc_prune_full - every option at once: gmc_prune_views plus multi-image
 * prompts.  image_id [B][N] int32 (device) gives each visual token's image,
 * ids 0..n_images-1 with every id present in every problem; NULL (or
 * n_images = 1) means one image.  With I = n_images > 1 (Sec. 3.1 totality
 * rule; App. H "Batched complementary support", "Appearance and spatial
 * clients"; Eq. cond-aux-clients; Eq. cond-assignment):
 *   - the realised budget is K = min{N, max{K_r, I}} (gmc_realized_budget);
 *   - the support starts with one token per image, the one of largest
 *     singleton gain F({i}) (ties to the lower index), then the batched
 *     rounds run until |S| = K (ceil((K - I) / b) rounds);
 *   - appearance clients cover their own image's tokens, and every image has
 *     its own L x L spatial landmarks on its own grid (M_S = L^2 I rows);
 *   - each token is assigned among its own image's carriers, and the gap
 *     delta is 0 for a token whose image has one carrier.
 * Multi-image calls use the exact appearance bank (N <= bounded_threshold_n,
 * else GMC_ERR_ARG).  Ids outside [0, I) are clamped and an image without
 * tokens gets the lowest unselected token as its seed; both are reported by
 * the GMC_STATUS_INPUT bit.  Other arguments as gmc_prune_views.
 * Errors: as gmc_prune_views; GMC_ERR_CAPACITY for I above max_images.
 */
#define GMC_MAX_IMAGES 64
#define GMC_STATUS_INPUT 8u   /* image ids out of range or an image without tokens */
int gmc_prune_full(int64_t B, const void* hidden, const void* text_q, const void* vis_k, const int32_t* pos3d,
                   const int32_t* image_id, int64_t n_images, int64_t N, int64_t T, int64_t K, void* out_hidden,
                   int32_t* out_pos, int32_t* out_idx, const float* nonvis_lse, int64_t n_hist,
                   const gmc_view* hist, const gmc_trace* trace);

/*
 * gmc_audit_message - the signed-message realisation audit of a compact
 * sequence (App. G Eq. cond-message-error; App. I Eq.
 * cond-message-decomposition, Eq. cond-softmax-bound, Eq.
 * cond-message-polar; Prop. 2 Eq. message-bound).  For every query/head
 * client g = (h, t) it re-runs native attention over the Full visual keys
 * and values and over the compact ones at the K carriers, both with the same
 * nonvisual log-sum-exp, and measures the signed messages y_g and y~_g, the
 * grouped Full mass M_gj over each carrier's cluster, the exact
 * decomposition y - y~ = term1 + term2 with term1 = sum_i a_gi (v_i -
 * v~_pi(i)) and term2 = sum_j (M_gj - abar_gj) v~_j, the grouped-mass gap
 * l1 = ||M_g - abar_g||_1 and its softmax contraction bound
 * max_j |u^F_gj - u^S_gj|.  Device pointers (dtype as the context's):
 *   text_q  [B][T][Hq][dh]; vis_k, vis_v [B][N][Hkv][dh] the Full visual
 *   keys and values of the next block; comp_k, comp_v [B][K][Hkv][dh] the
 *   keys and values of the compact visual tokens (the transported states at
 *   the carriers, in slot order); carrier [B][N] int32 each token's carrier
 *   slot in [0, K) (clamped); weights [B][Hq][T] fp32 client weights or NULL
 *   (uniform); nonvis_lse [B][Hq][T] fp32 or NULL.
 *   rows_out [B][Hq][T][GMC_AUDIT_ROW] fp32 or NULL: ||y||^2, ||y~||^2,
 *            <y, y~>, ||y - y~||^2, ||term1||^2, ||term2||^2, l1, bound
 *   vec_out  [B][Hq][T][4][dh] fp32 or NULL: y, y~, term1, term2
 *   out      [B][GMC_AUDIT_OUT] fp32: e_M = ||Y - Y~|| / (||Y|| + 1e-8),
 *            alpha = ||Y~|| / ||Y||, kappa = cos(Y, Y~), ||Y||, ||Y~||,
 *            ||Y - Y~||, max_g (l1 - bound) (<= 0 when the bound holds), 0;
 *            Y stacks sqrt(w_g) y_g.
 * A carrier slot without members has M_gj = 0 and an infinite bound.  With
 * gmc_prune's outputs, slot j is the j-th entry of out_idx and a token's
 * slot is the position of its traced carrier in out_idx.  Scratch comes from
 * the context's client-matrix buffer (the last call's client matrix is
 * overwritten; its outputs and diagnostics are kept).  Asynchronous on the
 * context's stream and ordered with the pruning calls like they are with
 * each other; nothing is allocated.
 * Errors: GMC_ERR_STATE, GMC_ERR_ARG, GMC_ERR_CAPACITY (scratch beyond the
 * client-matrix buffer), GMC_ERR_HIP.
 */
#define GMC_AUDIT_ROW 8
#define GMC_AUDIT_OUT 8
int gmc_audit_message(int64_t B, int64_t N, int64_t T, int64_t K, const void* text_q, const void* vis_k,
                      const void* vis_v, const void* comp_k, const void* comp_v, const int32_t* carrier,
                      const float* weights, const float* nonvis_lse, float* rows_out, float* vec_out, float* out);

/* Realised budget K = min{N, max{K_r, I}} for I images (Sec. 3.1); 0 if N < 1
 * or I < 1.  Host-only. */
int64_t gmc_realized_budget(int64_t N, int64_t K_req, int64_t n_images);

/*
 * Per-problem trace sizes of a gmc_prune_full call shape: selection rounds
 * (after the image seeds), pool capacity, batch capacity and client rows M
 * (every view's grounded rows, appearance, L^2 I spatial rows).
 */
int gmc_trace_dims_full(int64_t N, int64_t T, int64_t K, int64_t n_hist, int64_t n_images, int64_t* rounds,
                        int64_t* pool_cap, int64_t* batch_cap, int64_t* m_rows);

/* Realised budget K = min{N, max{K_r, 1}} (Sec. 3.1); 0 if N < 1. Host-only. */
int64_t gmc_realized_k(int64_t N, int64_t K_req);

/*
 * Per-problem trace sizes for a call shape under the current context:
 * selection rounds, pool capacity, batch capacity and client rows M.
 * Errors: GMC_ERR_STATE, GMC_ERR_ARG.  Host-only.
 */
int gmc_trace_dims(int64_t N, int64_t T, int64_t K, int64_t* rounds, int64_t* pool_cap,
                   int64_t* batch_cap, int64_t* m_rows);

/*
 * Stage timing for measurement.  While enabled, every subsequent call records
 * hipEvents on the context stream around each stage's launches, and all
 * stages run on that one stream (normally the bank kernels overlap the
 * message kernels on an internal stream), so each span times one stage:
 *   [0] row norms + value probe + mass coordinate   [1] message logits/softmax
 *   [2] head-pattern Gram + head weights + energy  [3] appearance bank GEMM
 *   [4] spatial bank + bank weights                [5] coverage refresh
 *   [6] singleton gains + candidate pool           [7] responsibility + batch
 *   [8] final coverage + objective values          [9] assignment
 *   [10] transport + compaction                    [11] per-call reset + row norms
 *   [12] persistent selection (all rounds in one launch; stages 5-7 and the
 *        final coverage are then empty)
 * gmc_timing_read synchronises the stream, returns per-stage total
 * milliseconds and span counts accumulated since the last read, and clears
 * them.  Errors: GMC_ERR_STATE, GMC_ERR_ARG (n < GMC_TIMERS), GMC_ERR_HIP.
 */
#define GMC_TIMERS 13
int gmc_timing_enable(int enable);
int gmc_timing_read(double* total_ms, int64_t* spans, int32_t n);

/*
 * Sequence compaction after pruning (App. H "Index map and physical token
 * accounting"; the cached deployment gathers prompt K/V of the prefix layers
 * at the retained sequence indices).  B sequences of L positions each hold
 * their N visual tokens at [vis_start, vis_start + N); out_idx [B][K] int32
 * (device) holds the K retained visual tokens of each, strictly ascending in
 * [0, N), as gmc_prune returns them.  The compacted length is
 * L2 = L - N + K, and position i maps to iota(i): unchanged before the visual
 * span, vis_start + k for the k-th retained visual token, i - (N - K) after
 * the span, -1 for a deleted visual position (order preserving).
 *
 * gmc_compact_sequence - for every sequence: (all device pointers, [B] leading)
 *   iota     [B][L]   int32 out, or NULL: the map above
 *   keep     [B][L2]  int32 out, or NULL: the retained original positions
 *            (the inverse map), the index list gmc_gather_rows takes
 *   seq_rows [B][L][row_bytes] in, out_rows [B][L2][row_bytes] out, vis_rows
 *            [B][K][row_bytes] in (the transported states, e.g. gmc_prune's
 *            out_hidden), all NULL or all set: text positions keep their
 *            row, the k-th retained visual position receives vis_rows row k
 *   seq_pos  [B][L][3] int32 in, out_pos [B][L2][3] int32 out, both NULL or
 *            both set: every retained position keeps its original ids
 * row_bytes is a positive multiple of 16, rows 16-byte aligned; 0 <= vis_start,
 * vis_start + N <= L, 1 <= K <= N.  out_idx entries that are not strictly
 * ascending in [0, N) give unspecified (but in-bounds) results.  Outputs
 * must not overlap inputs.  Runs on the context stream; needs a context (the
 * workspace is not used).  Errors: GMC_ERR_ARG, GMC_ERR_STATE, GMC_ERR_HIP.
 */
int gmc_compact_sequence(int64_t B, int64_t L, int64_t vis_start, int64_t N, int64_t K,
                         const int32_t* out_idx, int32_t* iota, int32_t* keep, const void* seq_rows,
                         const void* vis_rows, void* out_rows, int64_t row_bytes, const int32_t* seq_pos,
                         int32_t* out_pos);

/*
 * gmc_gather_rows - gather the rows of n_tensors caches at retained original
 * positions: dst[t][s][j] = src[t][s][keep[s / seqs_per_keep][j]] for every
 * tensor t < n_tensors, sequence s < n_seq and j < L2, rows of row_bytes
 * bytes.  src and dst are host arrays of n_tensors device pointers, each
 * tensor laid out [n_seq][L][row_bytes] (source) and [n_seq][L2][row_bytes]
 * (destination); seqs_per_keep consecutive sequences share one keep list
 * (keep [n_seq / seqs_per_keep][L2] int32, device, entries in [0, L)), e.g.
 * the heads of a head-major [B][Hkv][L][dh] cache with seqs_per_keep = Hkv,
 * or 1 for a token-major [B][L][Hkv * dh] cache.  1 <= n_tensors <= 64,
 * 1 <= n_seq <= 65535 a multiple of seqs_per_keep, row_bytes a positive multiple of 16,
 * rows 16-byte aligned.  Keep entries outside [0, L) are clamped.  Runs on
 * the context stream.  Errors: GMC_ERR_ARG, GMC_ERR_STATE, GMC_ERR_HIP.
 */
#define GMC_MAX_GATHER_TENSORS 64
int gmc_gather_rows(int64_t n_tensors, const void* const* src, void* const* dst, int64_t n_seq,
                    int64_t seqs_per_keep, int64_t L, int64_t L2, int64_t row_bytes, const int32_t* keep);

/*
 * gmc_prune_static - gmc_prune_ex without a context and without any device
 * allocation, for callers that cannot allocate device memory at call time:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation.  The workspace is carved, for this call's own shape, out of a
 * file-scope device array of GMC_STATIC_SCRATCH_BYTES per device (present
 * for the process's lifetime on every device the library runs on; its
 * address is looked up on the first call on a device).  Enough for one
 * problem at the Qwen2.5-VL-7B shape (N = 1296, T = 64, d = 3584, 28 / 4
 * heads, K = 256: about 23 MB).
 *   cfg      shape, settings and the value_probe / app_projection /
 *            value_probe_bias pointers as for gmc_init; its capacity fields are
 *            ignored (the call's B, N, T, K are the capacity)
 *   B, ..., nonvis_lse   as gmc_prune_ex (no trace)
 *   stream   hipStream_t for all work (NULL: the null stream); one stream,
 *            no side stream
 * Every call on a device shares that device's array and clears the region it
 * uses first: calls that overlap on one device race and give wrong results.
 * No diagnostics (gmc_get_diag reports on context calls only).  Errors:
 * GMC_ERR_ARG, GMC_ERR_CAPACITY (the call's workspace exceeds the array;
 * nothing is enqueued), GMC_ERR_HIP.
 */
#define GMC_STATIC_SCRATCH_BYTES (64ull << 20)
int gmc_prune_static(const gmc_config* cfg, int64_t B, const void* hidden, const void* text_q, const void* vis_k,
                     const int32_t* pos3d, int64_t N, int64_t T, int64_t K, void* out_hidden, int32_t* out_pos,
                     int32_t* out_idx, const float* nonvis_lse, void* stream);

/* Bytes of device workspace the current context holds (0 without one). */
int64_t gmc_workspace_bytes(void);

/* Description of the last error on this process (static storage). */
const char* gmc_last_error(void);

/* Release the context and its workspace; safe to call repeatedly. */
void gmc_free(void);

#ifdef __cplusplus
}
#endif

#endif /* GMC_H */
