// Message side of the GMC operator (Sec. 3.2; App. H "Native message
// clients"): row statistics, the folded value probe and mass coordinate
// (Eq. cond-mass-coordinate), the native text-query -> visual-key softmax
// slice with grounded atom energies (Eq. cond-native-message, Eq.
// cond-grounded-client), head-pattern Gram and farthest-first head weights
// (Eq. cond-head-pattern, Eq. cond-head-weight), and normalised grounded
// energy (Eq. cond-grounded-energy).
#include "gmc_device.h"
#include "gmc_gemm.h"
#include "gmc_internal.h"
#include "gmc_kernels.h"

namespace gmc {

// ---------------------------------------------------------------------------
// Squared row norms of the hidden states (one wave per token); the same
// kernel resets the per-call state, being the first of every call.
// ---------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256) rownorm_kernel(Shape sh, Ws ws, const T* hidden, int call_tag, int reset) {
  const int p = blockIdx.y;
  // the call's first kernel also resets the per-call state (a historical
  // view's states are normed later, into their own buffer, without it)
  if (reset) call_init_range(sh, ws, p, blockIdx.x * 256 + threadIdx.x, gridDim.x * 256);
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (i < sh.N) {
  const T* row = hidden + (static_cast<long long>(p) * sh.N + i) * sh.d;
  float s = 0.f;
#pragma unroll 4
  for (int k = lane * 8; k < sh.d; k += 64 * 8) {
    const uint4 raw = ld16(row + k);
    if constexpr (sizeof(T) == 2) {
      const bf16_t* v = reinterpret_cast<const bf16_t*>(&raw);
#pragma unroll
      for (int j = 0; j < 8; ++j) { const float f = bf16_to_f32(v[j]); s += f * f; }
    } else {
      const float* v = reinterpret_cast<const float*>(&raw);
#pragma unroll
      for (int j = 0; j < 4; ++j) s += v[j] * v[j];
      const uint4 raw2 = ld16(row + k + 4);
      const float* v2 = reinterpret_cast<const float*>(&raw2);
#pragma unroll
      for (int j = 0; j < 4; ++j) s += v2[j] * v2[j];
    }
  }
  s = wave_sum(s);
  // written through: the bank stream reads the norms without a kernel
  // boundary in between
  if (lane == 0) __hip_atomic_store(&ws.n2[p * ws.s_n + i], s, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  if (call_tag != 0) {
    // this block is done (its written-through stores have completed): tag it
    // with the call number for the bank stream's gate
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0)
      __hip_atomic_store(&ws.ftag[p * ws.s_ftag + blockIdx.x], call_tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// The bank stream's first kernel: one block waits until every row-norm block
// of the call has tagged itself, so the bank kernels that follow on that
// stream see the norms and the per-call reset, and start only after the
// caller's stream has finished the previous call.  The caller may have queued
// other work ahead of the call, so the wait is bounded in time (10 s of the
// constant clock), not in polls; a timeout raises the sticky status bit.
__global__ void __launch_bounds__(256) bank_gate_kernel(Shape sh, Ws ws, int call_tag) {
  const int nb = (sh.N + 3) / 4, total = nb * sh.B;
  const unsigned long long t0 = static_cast<unsigned long long>(wall_clock64());
  bool expired = false;
  for (int x0 = 0; x0 < total && !expired; x0 += 256 * 8) {
    int v[8];
    bool need[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int x = x0 + q * 256 + static_cast<int>(threadIdx.x);
      need[q] = x < total;
      const int xc = min(x, total - 1), p = xc / nb, b = xc % nb;
      v[q] = __hip_atomic_load(&ws.ftag[p * ws.s_ftag + b], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    for (int spin = 0;; ++spin) {
      bool pend = false;
#pragma unroll
      for (int q = 0; q < 8; ++q) pend |= need[q] && v[q] != call_tag;
      if (!pend) break;
      if ((spin & 255) == 255 && static_cast<unsigned long long>(wall_clock64()) - t0 > kGateWaitTicks) {
        raise_status(ws.cnt, kStatusBank);
        expired = true;
        break;
      }
      __builtin_amdgcn_s_sleep(8);   // a light poll: it may wait through a whole selection
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        if (!need[q] || v[q] == call_tag) continue;
        const int x = x0 + q * 256 + static_cast<int>(threadIdx.x), p = x / nb, b = x % nb;
        v[q] = __hip_atomic_load(&ws.ftag[p * ws.s_ftag + b], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
}

// Probe GEMM epilogue: Z[i][c] = (h_i . G_c) / sqrt(mean h_i^2 + eps), the
// folded value path applied to the next block's RMSNorm of h_i.
// Value probe partials: split s of problem p (combined index p * S + s)
// writes its K-slice of x_i . G[h][c] (the RMS scale is applied after the
// splits are summed).
struct ProbeSplitEpi {
  Ws ws;
  int hr;
  long long slot;    // N * hr floats per (problem, split)
  static constexpr bool kRowStats = false;
  __device__ float row_scale(int, int) const { return 1.f; }
  __device__ float col_scale(int, int) const { return 1.f; }
  __device__ float value(int pe, int r, int c, float v) const {
    ws.zp[static_cast<long long>(pe) * slot + static_cast<long long>(r) * hr + c] = v;
    return v;
  }
  __device__ void row_stats(int, int, int, float, float) const {}
};

// Z_h[i] = rms(h_i)^-1 sum_s partial_s (the next block's RMSNorm, unit gain)
// plus the folded value bias b_h when one is configured, and q_h[i] = ||Z_h[i]||^2, stored in place of the atom norm: consumers form
// l_h[i] = ||[Z_h[i]; sigma_h]|| = sqrt(q_h[i] + sigma_h^2).  One wave per
// (head, 64 tokens), lane = token; per-(block, head) sums of q are left for
// sigma_h = sqrt(lambda) max(sqrt(sum q / (N r)), eps), which the first
// block of the next kernel forms (sigma_from_partials).
// sigma_h from the per-(token block, head) sums of q, in token-block order.
__device__ void sigma_from_partials(const Shape& sh, const Params& pr, const Ws& ws, int p) {
  if (threadIdx.x >= sh.hq) return;
  const int hh = threadIdx.x, nb = (sh.N + 63) / 64;
  const float* part = ws.gpart + p * ws.s_gpart;
  float sum = 0.f;
  for (int b0 = 0; b0 < nb; b0 += 16) {
    float t[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) t[k] = part[min(b0 + k, nb - 1) * sh.hq + hh];
#pragma unroll
    for (int k = 0; k < 16; ++k)
      if (b0 + k < nb) sum += t[k];
  }
  const float mean2 = sum / (static_cast<float>(sh.N) * sh.r);
  ws.sig[p * ws.s_sig + hh] = sqrtf(pr.lambda_mass) * fmaxf(sqrtf(mean2), pr.eps_mass);
}

__global__ void __launch_bounds__(256) sigma_ell_kernel(Shape sh, Params pr, Ws ws, int ksplit) {
  const int p = blockIdx.z, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int h = blockIdx.y * 4 + wave;
  const int i = blockIdx.x * 64 + lane;
  float* part = ws.gpart + p * ws.s_gpart;          // free until the head-pattern Gram
  if (h < sh.hq) {
    const int ic = min(i, sh.N - 1);
    const float* zp = ws.zp + static_cast<long long>(p) * ksplit * sh.N * sh.hr +
                      static_cast<long long>(ic) * sh.hr + h * sh.r;
    const long long sstride = static_cast<long long>(sh.N) * sh.hr;
    float v[kProbeSplit][kMaxProbe];
#pragma unroll
    for (int s = 0; s < kProbeSplit; ++s)
#pragma unroll
      for (int c = 0; c < kMaxProbe; ++c)
        v[s][c] = (s < ksplit && c < sh.r) ? zp[s * sstride + c] : 0.f;
    const float rs = rsqrtf(ws.n2[p * ws.s_n + ic] / static_cast<float>(sh.d) + pr.rms_eps);
    float q = 0.f;
    float* z = ws.z + p * ws.s_z + static_cast<long long>(ic) * sh.hr + h * sh.r;
#pragma unroll
    for (int c = 0; c < kMaxProbe; ++c) {
      if (c < sh.r) {
        const float zs = (((v[0][c] + v[1][c]) + v[2][c]) + v[3][c]) * rs;
        const float zc = pr.probe_bias ? zs + pr.probe_bias[h * sh.r + c] : zs;
        q += zc * zc;
        if (i < sh.N) z[c] = zc;
      }
    }
    if (i < sh.N) ws.ell[p * ws.s_ell + static_cast<long long>(h) * sh.N + i] = q;
    const float bq = wave_sum(i < sh.N ? q : 0.f);
    if (lane == 0) part[blockIdx.x * sh.hq + h] = bq;
  }
}

// ---------------------------------------------------------------------------
// Native message slice and grounded energies.
// A block covers 16 rows (h,t) of one kv group and one of lsplit column
// ranges; its waves take the 16-column tiles of the range in turn.  Two
// kernels: logits_lse_kernel reduces the online max / sum-exp of the logits
// q.k/sqrt(dh) over the block's columns into per-range partials;
// logits_kernel combines the partials into the log-sum-exp D (optionally
// extended by the nonvisual part), recomputes the logits (cheaper than
// storing them), writes e = exp(s - D) l_h[i] to the grounded client rows and
// leaves per-range row sums and row maxima.  Nothing but e reaches HBM.
// Splitting the columns over blocks puts every CU to work on the key stream.
// These generic kernels serve fp32, wide heads and query counts that are not
// a multiple of 16; bf16 calls use the staged pair below (or, while one
// 16-row block per CU suffices, the register kernel).
// ---------------------------------------------------------------------------
// Waves per logits block, each on its own key tiles (fewer where the fp32
// fragments of a wide head would not fit the registers of eight waves).
template <typename T, int DH>
constexpr int logit_waves() { return (sizeof(T) == 4 && DH >= 224) ? 4 : 8; }

// Tiles per wave and chunk: every load of a chunk is issued before its first
// MFMA, so a chunk costs one memory latency and no load is in flight across
// the chunk loop's back edge (where the compiler would wait for everything).
template <typename T, int DH>
constexpr int logit_chunk() {
  constexpr int KS = DH / 32, FR = static_cast<int>(sizeof(Frag<T>) / 4);
  constexpr int budget = logit_waves<T, DH>() == 4 ? 192 : 96;   // registers for key tiles
  return budget / (KS * FR) < 1 ? 1 : (budget / (KS * FR) > 6 ? 6 : budget / (KS * FR));
}

// Shared set-up of both logits kernels: block coordinates, the query
// fragments (A operand, row rb + fr), key addressing and the column range.
template <typename T, int DH>
struct LogitBlock {
  static constexpr int KS = DH / 32;
  int p, g, rb, split, rows_g, t_beg, t_end;
  int lane, wave, fr, fk, orow, oc;
  float scale;
  const T* kbase;
  long long kstride;
  Frag<T> qf[KS];

  __device__ LogitBlock(const Shape& sh, const T* text_q, const T* vis_k, int lsplit) {
    p = blockIdx.z;
    g = blockIdx.y;
    rb = (blockIdx.x / lsplit) * 16;
    split = blockIdx.x % lsplit;
    rows_g = sh.hg * sh.T;
    lane = threadIdx.x & 63;
    wave = wave_id();
    fr = lane & 15;
    fk = (lane >> 4) * 8;
    orow = (lane >> 4) * 4;
    oc = lane & 15;
    scale = rsqrtf(static_cast<float>(DH));
    const int ntile = (sh.N + 15) / 16, tps = (ntile + lsplit - 1) / lsplit;
    t_beg = min(ntile, split * tps);
    t_end = min(ntile, t_beg + tps);
    const int rr = rb + fr;
    if (rr < rows_g) {
      const int h = g * sh.hg + rr / sh.T, t = rr % sh.T;
      const T* q = text_q + ((static_cast<long long>(p) * sh.T + t) * sh.hq + h) * DH;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qf[ks] = frag_load<T>(q + ks * 32 + fk);
    } else {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qf[ks] = frag_zero<T>();
    }
    kbase = vis_k + static_cast<long long>(p) * sh.N * sh.hkv * DH + g * DH;
    kstride = static_cast<long long>(sh.hkv) * DH;
  }
  // key fragments of a column tile; the column is clamped so the loads are
  // unconditional (out-of-range columns are masked by the callers)
  __device__ void load_keys(const Shape& sh, int ct, Frag<T>* kf) const {
    const int col = min(ct * 16 + fr, sh.N - 1);
    const T* kr = kbase + col * kstride;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) kf[ks] = frag_load<T>(kr + ks * 32 + fk);
  }
  __device__ floatx4 tile_mma(const Frag<T>* kf) const {
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) acc = mma(qf[ks], kf[ks], acc);
    return acc;
  }
  // grounded client row of block row r (valid rows only)
  __device__ long long mrow(const Shape& sh, int r) const {
    const int rr = rb + r;
    return static_cast<long long>(g * sh.hg + rr / sh.T) * sh.T + rr % sh.T;
  }
};

template <typename T, int DH>
__global__ void __launch_bounds__((64 * logit_waves<T, DH>()))
logits_lse_kernel(Shape sh, Params pr, Ws ws, const T* text_q, const T* vis_k) {
  constexpr int W = logit_waves<T, DH>(), MT = logit_chunk<T, DH>(), KS = DH / 32;
  __shared__ float sm_m[W][16], sm_s[W][16];
  const LogitBlock<T, DH> lb(sh, text_q, vis_k, sh.lsplit);
  // online (max, sum exp) per row, lane-local over its columns
  float mx[4], sm[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) { mx[e] = -INFINITY; sm[e] = 0.f; }
  for (int c0 = lb.t_beg + lb.wave; c0 < lb.t_end; c0 += MT * W) {
    Frag<T> kf[MT][KS];
#pragma unroll
    for (int j = 0; j < MT; ++j)
      if (c0 + j * W < lb.t_end) lb.load_keys(sh, c0 + j * W, kf[j]);
#pragma unroll
    for (int j = 0; j < MT; ++j) {
      const int ct = c0 + j * W;
      if (ct < lb.t_end) {
        const floatx4 acc = lb.tile_mma(kf[j]);
        if (ct * 16 + lb.oc < sh.N) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float s = acc[e] * lb.scale;
            const float nm = fmaxf(mx[e], s);
            sm[e] = sm[e] * __expf(mx[e] - nm) + __expf(s - nm);
            mx[e] = nm;
          }
        }
      }
    }
  }
  // merge across the 16 lanes of a row group (maximum first, then each
  // lane's sum rescaled once and added), then across waves
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float m = group16_max(mx[e]);
    const float sc = (mx[e] == -INFINITY) ? 0.f : sm[e] * __expf(mx[e] - m);
    const float t = group16_sum(sc);
    if (lb.oc == 0) { sm_m[lb.wave][lb.orow + e] = m; sm_s[lb.wave][lb.orow + e] = t; }
  }
  __syncthreads();
  if (threadIdx.x < 16) {
    const int r = threadIdx.x;
    if (lb.rb + r < lb.rows_g) {
      float m = -INFINITY;
      for (int w = 0; w < W; ++w) m = fmaxf(m, sm_m[w][r]);
      float s = 0.f;
      for (int w = 0; w < W; ++w) s += (sm_m[w][r] == -INFINITY) ? 0.f : sm_s[w][r] * __expf(sm_m[w][r] - m);
      float* part = ws.lpart + lb.p * ws.s_lpart;
      const long long mi = lb.mrow(sh, r);
      part[static_cast<long long>(lb.split) * sh.mg + mi] = m;
      part[static_cast<long long>(kLogitSplit + lb.split) * sh.mg + mi] = s;
    }
  }
  // one spare job for the problem's first block: the mass coordinates, needed
  // from the next kernel on
  if (blockIdx.x == 0 && blockIdx.y == 0) sigma_from_partials(sh, pr, ws, lb.p);
}

template <typename T, int DH>
__global__ void __launch_bounds__((64 * logit_waves<T, DH>()))
logits_kernel(Shape sh, Ws ws, const T* text_q, const T* vis_k, const float* nonvis_lse) {
  constexpr int W = logit_waves<T, DH>(), MT = logit_chunk<T, DH>(), KS = DH / 32;
  __shared__ float sm_m[W][16], sm_s[W][16];
  __shared__ float sm_D[16];
  const LogitBlock<T, DH> lb(sh, text_q, vis_k, sh.lsplit);
  float* part = ws.lpart + lb.p * ws.s_lpart;
  if (threadIdx.x < 16) {
    // the row's log-sum-exp from the per-range partials, in range order
    const int r = threadIdx.x, rr = lb.rb + r;
    float D = 0.f;
    if (rr < lb.rows_g) {
      const long long mi = lb.mrow(sh, r);
      float m = -INFINITY;
      for (int s = 0; s < sh.lsplit; ++s) m = fmaxf(m, part[static_cast<long long>(s) * sh.mg + mi]);
      float sum = 0.f;
      for (int s = 0; s < sh.lsplit; ++s) {
        const float ms = part[static_cast<long long>(s) * sh.mg + mi];
        sum += (ms == -INFINITY) ? 0.f : part[static_cast<long long>(kLogitSplit + s) * sh.mg + mi] * expf(ms - m);
      }
      D = m + logf(sum);
      if (nonvis_lse) {
        const int h = lb.g * sh.hg + rr / sh.T, t = rr % sh.T;
        const float nv = nonvis_lse[(static_cast<long long>(lb.p) * sh.hq + h) * sh.T + t];
        const float hi = fmaxf(D, nv), lo = fminf(D, nv);
        D = (hi == -INFINITY) ? hi : hi + log1pf(expf(lo - hi));
      }
    }
    sm_D[r] = D;
  }
  __syncthreads();

  // e = A * l, written to the grounded client rows; row sums / maxima
  float D[4], rsum[4], rmax[4], sig2[4];
  int hrow[4];
  long long mrow[4];
  bool rvalid[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int rr = lb.rb + lb.orow + e;
    rvalid[e] = rr < lb.rows_g;
    hrow[e] = lb.g * sh.hg + (rvalid[e] ? rr / sh.T : 0);
    mrow[e] = rvalid[e] ? lb.mrow(sh, lb.orow + e) : 0;
    D[e] = sm_D[lb.orow + e];
    rsum[e] = 0.f;
    rmax[e] = 0.f;
    const float sg = ws.sig[lb.p * ws.s_sig + hrow[e]];
    sig2[e] = sg * sg;
  }
  // with T a multiple of 16 the 16 rows of a block are one head's
  // consecutive queries: a lane's four rows are four consecutive client rows
  // (one 16-byte store per tile) and share the atom norm l_h[col]
  const bool vec = (sh.T & 15) == 0;
  float* E = ws.E + lb.p * ws.s_E;
  const float* ell = ws.ell + lb.p * ws.s_ell;
  for (int c0 = lb.t_beg + lb.wave; c0 < lb.t_end; c0 += MT * W) {
    Frag<T> kf[MT][KS];
    float lv[MT][4];
#pragma unroll
    for (int j = 0; j < MT; ++j) {
      const int ct = c0 + j * W;
      if (ct >= lb.t_end) continue;
      lb.load_keys(sh, ct, kf[j]);
      const int col = min(ct * 16 + lb.oc, sh.N - 1);
      if (vec) {
        lv[j][0] = ell[static_cast<long long>(hrow[0]) * sh.N + col];
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) lv[j][e] = ell[static_cast<long long>(hrow[e]) * sh.N + col];
      }
    }
#pragma unroll
    for (int j = 0; j < MT; ++j) {
      const int ct = c0 + j * W;
      if (ct >= lb.t_end) continue;
      const floatx4 acc = lb.tile_mma(kf[j]);
      const int col = ct * 16 + lb.oc;
      if (col >= sh.N) continue;
      float v[4];
      // atom norm l_h[col]: one per column when the lane's four rows share the head
      const float nrm0 = vec ? sqrtf(lv[j][0] + sig2[0]) : 0.f;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float a = __expf(acc[e] * lb.scale - D[e]);
        v[e] = a * (vec ? nrm0 : sqrtf(lv[j][e] + sig2[e]));
      }
      if (vec) {
        *reinterpret_cast<float4*>(E + static_cast<long long>(col) * sh.ldM + mrow[0]) =
            make_float4(v[0], v[1], v[2], v[3]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          rsum[e] += v[e];
          rmax[e] = fmaxf(rmax[e], v[e]);
        }
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (!rvalid[e]) continue;
          E[static_cast<long long>(col) * sh.ldM + mrow[e]] = v[e];
          rsum[e] += v[e];
          rmax[e] = fmaxf(rmax[e], v[e]);
        }
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float s = group16_sum(rsum[e]);
    const float m = group16_max(rmax[e]);
    if (lb.oc == 0) { sm_s[lb.wave][lb.orow + e] = s; sm_m[lb.wave][lb.orow + e] = m; }
  }
  __syncthreads();
  const int r = threadIdx.x;
  const bool row = r < 16 && lb.rb + r < lb.rows_g;
  const long long mi = row ? lb.mrow(sh, r) : 0;
  float s = 0.f, m = 0.f;
  if (row)
    for (int w = 0; w < W; ++w) { s += sm_s[w][r]; m = fmaxf(m, sm_m[w][r]); }
  if (sh.lsplit == 1) {
    if (row) {
      ws.rowsum[lb.p * ws.s_m + mi] = s;
      ws.peak[lb.p * ws.s_m + mi] = m;   // max_i e; scaled by the row weight later
    }
    return;
  }
  // the last of the row tile's ranges adds the range partials in range order
  if (row) {
    st_dev(&part[static_cast<long long>(2 * kLogitSplit + lb.split) * sh.mg + mi], s);
    st_dev(&part[static_cast<long long>(3 * kLogitSplit + lb.split) * sh.mg + mi], m);
  }
  __shared__ int flag;
  int* cnt = ws.lcnt + lb.p * ws.s_lcnt + (blockIdx.x / sh.lsplit) * sh.hkv + lb.g;
  if (!last_arrival(cnt, sh.lsplit, &flag)) return;
  if (row) {
    // every load in flight first, then the sums in range order
    float vs[kLogitSplit], vm[kLogitSplit];
#pragma unroll
    for (int q = 0; q < kLogitSplit; ++q) {
      const int qc = min(q, sh.lsplit - 1);
      vs[q] = ld_dev(&part[static_cast<long long>(2 * kLogitSplit + qc) * sh.mg + mi]);
      vm[q] = ld_dev(&part[static_cast<long long>(3 * kLogitSplit + qc) * sh.mg + mi]);
    }
    float ts = 0.f, tm = 0.f;
#pragma unroll
    for (int q = 0; q < kLogitSplit; ++q)
      if (q < sh.lsplit) { ts += vs[q]; tm = fmaxf(tm, vm[q]); }
    ws.rowsum[lb.p * ws.s_m + mi] = ts;
    ws.peak[lb.p * ws.s_m + mi] = tm;
  }
  if (threadIdx.x == 0) st_dev(cnt, 0);
}

// Staged form of the column-range kernels (bf16, T a multiple of 16): a block
// of kStW waves covers 16 kStW consecutive rows of one kv group, one 16-row
// MFMA fragment (inside one head) per wave.  The block's key tiles pass
// through LDS in stages of kStSG tiles, double buffered (the next stage's
// global loads are in flight while the waves work on this one), so each key
// byte is read from L2 once per block and feeds every wave's fragment.
constexpr int kStW = 8;                   // waves per staged block
constexpr int kStRows = 16 * kStW;        // rows per staged block
constexpr int kStSG = 4;                  // key tiles per LDS stage
constexpr int kStPad = 8;                 // bf16 padding per staged key row (bank spread)

template <int DH>
struct StageBlock {
  static constexpr int KS = DH / 32;
  static constexpr int ROW = DH + kStPad;                                   // staged row, elements
  static constexpr int CPT = DH / 8;                                        // 16-byte chunks per key row
  static constexpr int NCH = kStSG * 16 * CPT;                              // chunks per stage
  static constexpr int CH = (NCH + 64 * kStW - 1) / (64 * kStW);           // chunks per thread
  static constexpr int BUF = kStSG * 16 * ROW;                              // elements per stage buffer
  int p, g, rb, split, rows_g, t_beg, t_end, nst;
  int lane, wave, fr, fk, orow, oc;
  bool active;     // the wave's fragment holds rows
  float scale;
  const bf16_t* kbase;
  long long kstride;
  Frag<bf16_t> qf[KS];

  __device__ StageBlock(const Shape& sh, const bf16_t* text_q, const bf16_t* vis_k, int lsplit) {
    p = blockIdx.z;
    g = blockIdx.y;
    rb = (blockIdx.x / lsplit) * kStRows;
    split = blockIdx.x % lsplit;
    rows_g = sh.hg * sh.T;                   // a multiple of 16
    lane = threadIdx.x & 63;
    wave = wave_id();
    fr = lane & 15;
    fk = (lane >> 4) * 8;
    orow = (lane >> 4) * 4;
    oc = lane & 15;
    active = rb + 16 * wave < rows_g;
    scale = rsqrtf(static_cast<float>(DH));
    const int ntile = (sh.N + 15) / 16, tps = (ntile + lsplit - 1) / lsplit;
    t_beg = min(ntile, split * tps);
    t_end = min(ntile, t_beg + tps);
    nst = (t_end - t_beg + kStSG - 1) / kStSG;
    if (active) {
      const int rr = rb + 16 * wave + fr;
      const int h = g * sh.hg + rr / sh.T, t = rr % sh.T;
      const bf16_t* q = text_q + ((static_cast<long long>(p) * sh.T + t) * sh.hq + h) * DH;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qf[ks] = frag_load<bf16_t>(q + ks * 32 + fk);
    } else {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qf[ks] = frag_zero<bf16_t>();
    }
    kbase = vis_k + static_cast<long long>(p) * sh.N * sh.hkv * DH + g * DH;
    kstride = static_cast<long long>(sh.hkv) * DH;
  }
  // this thread's 16-byte chunks of stage s (columns clamped to the last token)
  __device__ void stage_load(const Shape& sh, int s, uint4* r) const {
    const int c0 = (t_beg + s * kStSG) * 16;
#pragma unroll
    for (int q = 0; q < CH; ++q) {
      const int c = min(static_cast<int>(threadIdx.x) + q * 64 * kStW, NCH - 1);
      const int col = min(c0 + c / CPT, sh.N - 1);
      r[q] = ld16(kbase + col * kstride + (c % CPT) * 8);
    }
  }
  __device__ void stage_store(bf16_t* buf, const uint4* r) const {
#pragma unroll
    for (int q = 0; q < CH; ++q) {
      const int c = threadIdx.x + q * 64 * kStW;
      if (c < NCH) st16(buf + (c / CPT) * ROW + (c % CPT) * 8, r[q]);
    }
  }
  // the wave's 16 x 16 logit tile against key tile j of a staged buffer
  __device__ floatx4 tile_mma(const bf16_t* buf, int j) const {
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
    const bf16_t* kr = buf + (j * 16 + fr) * ROW + fk;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      Frag<bf16_t> kf;
      kf.v = __builtin_bit_cast(bf16x8, ld16(kr + ks * 32));
      acc = mma(qf[ks], kf, acc);
    }
    return acc;
  }
  // client row of the wave's fragment row 0 (rows of a group are consecutive client rows)
  __device__ long long mrow0(const Shape& sh) const { return static_cast<long long>(g) * rows_g + rb + 16 * wave; }
};

template <int DH>
__global__ void __launch_bounds__(64 * kStW)
logits_lse_stage_kernel(Shape sh, Params pr, Ws ws, const bf16_t* text_q, const bf16_t* vis_k) {
  using SB = StageBlock<DH>;
  __shared__ __attribute__((aligned(16))) bf16_t kst[2 * SB::BUF];
  const SB lb(sh, text_q, vis_k, sh.lsplit);
  // online (max, sum) per row in the base-2 domain (y = s log2 e): a lane's
  // sum is rescaled only when its running maximum grows
  const float c2 = lb.scale * 1.44269504088896341f;
  float mx[4], sm[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) { mx[e] = -INFINITY; sm[e] = 0.f; }
  uint4 rg[SB::CH];
  if (lb.nst > 0) lb.stage_load(sh, 0, rg);
  for (int s = 0; s < lb.nst; ++s) {
    bf16_t* buf = kst + (s & 1) * SB::BUF;
    lb.stage_store(buf, rg);
    __syncthreads();
    if (s + 1 < lb.nst) lb.stage_load(sh, s + 1, rg);
    if (lb.active) {
#pragma unroll
      for (int j = 0; j < kStSG; ++j) {
        const int ct = lb.t_beg + s * kStSG + j;
        if (ct >= lb.t_end) break;   // block-uniform
        const floatx4 acc = lb.tile_mma(buf, j);
        if (ct * 16 + lb.oc >= sh.N) continue;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float y = acc[e] * c2;
          if (y > mx[e]) {
            sm[e] *= __builtin_amdgcn_exp2f(mx[e] - y);
            mx[e] = y;
          }
          sm[e] += __builtin_amdgcn_exp2f(y - mx[e]);
        }
      }
    }
  }
  // merge across the 16 lanes of a row group; each wave owns its rows
  if (lb.active) {
    float* part = ws.lpart + lb.p * ws.s_lpart;
    const long long m0 = lb.mrow0(sh);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float m = group16_max(mx[e]);
      const float sc = (mx[e] == -INFINITY) ? 0.f : sm[e] * __builtin_amdgcn_exp2f(mx[e] - m);
      const float t = group16_sum(sc);
      if (lb.oc == 0) {
        const long long mi = m0 + lb.orow + e;
        part[static_cast<long long>(lb.split) * sh.mg + mi] = m * 0.69314718055994531f;
        part[static_cast<long long>(kLogitSplit + lb.split) * sh.mg + mi] = t;
      }
    }
  }
  // one spare job for the problem's first block: the mass coordinates, needed
  // from the next kernel on
  if (blockIdx.x == 0 && blockIdx.y == 0) sigma_from_partials(sh, pr, ws, lb.p);
}

template <int DH>
__global__ void __launch_bounds__(64 * kStW)
logits_stage_kernel(Shape sh, Ws ws, const bf16_t* text_q, const bf16_t* vis_k, const float* nonvis_lse) {
  using SB = StageBlock<DH>;
  __shared__ __attribute__((aligned(16))) bf16_t kst[2 * SB::BUF];
  __shared__ float sm_D[kStRows];
  const SB lb(sh, text_q, vis_k, sh.lsplit);
  float* part = ws.lpart + lb.p * ws.s_lpart;
  const long long mb = static_cast<long long>(lb.g) * lb.rows_g + lb.rb;   // client row of block row 0
  if (threadIdx.x < kStRows) {
    // the row's log-sum-exp from the per-range partials, in range order
    const int r = threadIdx.x, rr = lb.rb + r;
    float D = 0.f;
    if (rr < lb.rows_g) {
      const long long mi = mb + r;
      float m = -INFINITY;
      for (int s = 0; s < sh.lsplit; ++s) m = fmaxf(m, part[static_cast<long long>(s) * sh.mg + mi]);
      float sum = 0.f;
      for (int s = 0; s < sh.lsplit; ++s) {
        const float ms = part[static_cast<long long>(s) * sh.mg + mi];
        sum += (ms == -INFINITY) ? 0.f : part[static_cast<long long>(kLogitSplit + s) * sh.mg + mi] * expf(ms - m);
      }
      D = m + logf(sum);
      if (nonvis_lse) {
        const int h = lb.g * sh.hg + rr / sh.T, t = rr % sh.T;
        const float nv = nonvis_lse[(static_cast<long long>(lb.p) * sh.hq + h) * sh.T + t];
        const float hi = fmaxf(D, nv), lo = fminf(D, nv);
        D = (hi == -INFINITY) ? hi : hi + log1pf(expf(lo - hi));
      }
    }
    sm_D[r] = D;
  }
  __syncthreads();
  // e = A * l, written to the grounded client rows; row sums / maxima
  const float c2 = lb.scale * 1.44269504088896341f;
  const int h = lb.g * sh.hg + (lb.active ? (lb.rb + 16 * lb.wave) / sh.T : 0);   // the wave's head
  const float sg = ws.sig[lb.p * ws.s_sig + h];
  const float sig2 = sg * sg;
  float D2[4], rsum[4], rmax[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    D2[e] = sm_D[16 * lb.wave + lb.orow + e] * 1.44269504088896341f;
    rsum[e] = 0.f;
    rmax[e] = 0.f;
  }
  const long long m0 = lb.mrow0(sh);
  float* E = ws.E + lb.p * ws.s_E + m0 + lb.orow;
  const float* ellh = ws.ell + lb.p * ws.s_ell + static_cast<long long>(h) * sh.N;
  // the lane's atom norms l_h[col] of a stage (its column in each tile)
  auto norms = [&](int s, float* lv) {
#pragma unroll
    for (int j = 0; j < kStSG; ++j) lv[j] = ellh[min((lb.t_beg + s * kStSG + j) * 16 + lb.oc, sh.N - 1)];
  };
  uint4 rg[SB::CH];
  float lv[kStSG], lvn[kStSG];
  if (lb.nst > 0) {
    lb.stage_load(sh, 0, rg);
    norms(0, lvn);
  }
  for (int s = 0; s < lb.nst; ++s) {
    bf16_t* buf = kst + (s & 1) * SB::BUF;
    lb.stage_store(buf, rg);
#pragma unroll
    for (int j = 0; j < kStSG; ++j) lv[j] = lvn[j];
    __syncthreads();
    if (s + 1 < lb.nst) {
      lb.stage_load(sh, s + 1, rg);
      norms(s + 1, lvn);
    }
    if (lb.active) {
#pragma unroll
      for (int j = 0; j < kStSG; ++j) {
        const int ct = lb.t_beg + s * kStSG + j;
        if (ct >= lb.t_end) break;   // block-uniform
        const floatx4 acc = lb.tile_mma(buf, j);
        const int col = ct * 16 + lb.oc;
        if (col >= sh.N) continue;
        const float nrm = sqrtf(lv[j] + sig2);
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[e] = __builtin_amdgcn_exp2f(acc[e] * c2 - D2[e]) * nrm;
          rsum[e] += v[e];
          rmax[e] = fmaxf(rmax[e], v[e]);
        }
        *reinterpret_cast<float4*>(E + static_cast<long long>(col) * sh.ldM) = make_float4(v[0], v[1], v[2], v[3]);
      }
    }
  }
  // per-row sums and maxima (each wave owns its rows)
  float rs[4], rm[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    rs[e] = group16_sum(rsum[e]);
    rm[e] = group16_max(rmax[e]);
  }
  const bool wrote = lb.active && lb.oc == 0;
  if (sh.lsplit == 1) {
    if (wrote)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        ws.rowsum[lb.p * ws.s_m + m0 + lb.orow + e] = rs[e];
        ws.peak[lb.p * ws.s_m + m0 + lb.orow + e] = rm[e];   // max_i e; scaled by the row weight later
      }
    return;
  }
  // the last of the row block's ranges adds the range partials in range order
  if (wrote)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const long long mi = m0 + lb.orow + e;
      st_dev(&part[static_cast<long long>(2 * kLogitSplit + lb.split) * sh.mg + mi], rs[e]);
      st_dev(&part[static_cast<long long>(3 * kLogitSplit + lb.split) * sh.mg + mi], rm[e]);
    }
  __shared__ int flag;
  int* cnt = ws.lcnt + lb.p * ws.s_lcnt + (blockIdx.x / sh.lsplit) * sh.hkv + lb.g;
  if (!last_arrival(cnt, sh.lsplit, &flag)) return;
  const int r = threadIdx.x;
  if (r < kStRows && lb.rb + r < lb.rows_g) {
    const long long mi = mb + r;
    float vs[kLogitSplit], vm[kLogitSplit];
#pragma unroll
    for (int q = 0; q < kLogitSplit; ++q) {
      const int qc = min(q, sh.lsplit - 1);
      vs[q] = ld_dev(&part[static_cast<long long>(2 * kLogitSplit + qc) * sh.mg + mi]);
      vm[q] = ld_dev(&part[static_cast<long long>(3 * kLogitSplit + qc) * sh.mg + mi]);
    }
    float ts = 0.f, tm = 0.f;
#pragma unroll
    for (int q = 0; q < kLogitSplit; ++q)
      if (q < sh.lsplit) { ts += vs[q]; tm = fmaxf(tm, vm[q]); }
    ws.rowsum[lb.p * ws.s_m + mi] = ts;
    ws.peak[lb.p * ws.s_m + mi] = tm;
  }
  if (threadIdx.x == 0) st_dev(cnt, 0);
}

// Small N: a block keeps its 16 rows' logits over every column in registers
// (at most MAXT tiles per wave), so the keys are read once, the log-sum-exp is
// reduced inside the block, and e is written with 16-byte stores; the mass
// coordinates of the block's heads are formed from the probe partials first.
constexpr int kLogitRegTiles = 12;   // tiles per wave held in registers
// configurations whose query and key fragments leave room for the tiles
template <typename T, int DH>
constexpr bool logit_reg_ok() {
  return logit_waves<T, DH>() == 8 && (DH / 32) * static_cast<int>(sizeof(Frag<T>) / 4) <= 32;
}

// VEC (T a multiple of 16): the 16 rows of a block are one head's consecutive
// queries, so a lane's four rows share the head, its atom norms and sigma
// (one norm per column instead of four) and are four consecutive client rows
// (one 16-byte store per tile).
template <typename T, int DH, int MAXT, bool VEC>
__global__ void __launch_bounds__(512)
logits_reg_kernel(Shape sh, Params pr, Ws ws, const T* text_q, const T* vis_k, const float* nonvis_lse) {
  constexpr int W = 8, MT = logit_chunk<T, DH>(), KS = DH / 32;
  __shared__ float sm_m[W][16], sm_s[W][16], sm_D[16], sm_sig[16];
  const LogitBlock<T, DH> lb(sh, text_q, vis_k, 1);
  const int ntile = (sh.N + 15) / 16;
  // sigma of each block row's head (threads 0..15) and, in block (0, 0), of
  // every head for the head-pattern kernel (threads 64 + h): the partials of
  // the token blocks (at most 1536 / 64 on this path) go out now and are
  // added, in token-block order, after the logits
  constexpr int kSigB = 16 * 8 * MAXT / 64;
  const int nb = (sh.N + 63) / 64;
  const bool own_sig = threadIdx.x < 16;
  const bool all_sig = blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x >= 64 && threadIdx.x < 64 + sh.hq;
  float sg_t[kSigB];
  if (own_sig || all_sig) {
    const int rr = lb.rb + threadIdx.x;
    const int h = own_sig ? lb.g * sh.hg + (rr < lb.rows_g ? rr / sh.T : 0) : static_cast<int>(threadIdx.x) - 64;
    const float* part = ws.gpart + lb.p * ws.s_gpart;
#pragma unroll
    for (int k = 0; k < kSigB; ++k) sg_t[k] = part[min(k, nb - 1) * sh.hq + h];
  }

  int hrow[4];
  long long mrow[4];
  bool rvalid[4];
  if constexpr (VEC) {
    // one head per block: its index and the first query are block-uniform
    const int h = lb.g * sh.hg + lb.rb / sh.T, t0 = lb.rb % sh.T + lb.orow;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      rvalid[e] = lb.rb + lb.orow + e < lb.rows_g;
      hrow[e] = h;
      mrow[e] = static_cast<long long>(h) * sh.T + t0 + e;
    }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int rr = lb.rb + lb.orow + e;
      rvalid[e] = rr < lb.rows_g;
      hrow[e] = lb.g * sh.hg + (rvalid[e] ? rr / sh.T : 0);
      mrow[e] = rvalid[e] ? lb.mrow(sh, lb.orow + e) : 0;
    }
  }
  const float* ell = ws.ell + lb.p * ws.s_ell;
  // logits s = q.k / sqrt(dh) of the wave's tiles wave, wave + W, ...:
  // chunks of MT tiles, every load of a chunk before its MFMAs
  floatx4 sv[MAXT];
  float lv[MAXT][4];
#pragma unroll
  for (int c = 0; c < MAXT; c += MT) {
    Frag<T> kf[MT][KS];
#pragma unroll
    for (int j = 0; j < MT; ++j) {
      const int t = c + j, ct = lb.wave + t * W;
      if (t < MAXT && ct < ntile) {
        lb.load_keys(sh, ct, kf[j]);
        const int col = min(ct * 16 + lb.oc, sh.N - 1);
        if constexpr (VEC) {
          lv[t][0] = ell[static_cast<long long>(hrow[0]) * sh.N + col];
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) lv[t][e] = ell[static_cast<long long>(hrow[e]) * sh.N + col];
        }
      }
    }
#pragma unroll
    for (int j = 0; j < MT; ++j) {
      const int t = c + j, ct = lb.wave + t * W;
      if (t < MAXT) {
        const bool ok = ct < ntile && ct * 16 + lb.oc < sh.N;
        const floatx4 acc = ct < ntile ? lb.tile_mma(kf[j]) : floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int e = 0; e < 4; ++e) sv[t][e] = ok ? acc[e] * lb.scale : -INFINITY;
      }
    }
  }
  if (own_sig || all_sig) {
    float sum = 0.f;
#pragma unroll
    for (int k = 0; k < kSigB; ++k)
      if (k < nb) sum += sg_t[k];
    const float mean2 = sum / (static_cast<float>(sh.N) * sh.r);
    const float sg = sqrtf(pr.lambda_mass) * fmaxf(sqrtf(mean2), pr.eps_mass);
    if (own_sig) sm_sig[threadIdx.x] = sg;
    else ws.sig[lb.p * ws.s_sig + threadIdx.x - 64] = sg;
  }
  // log-sum-exp per row: lane, 16-lane group (maximum first), waves
  float mx[4], sm[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    float m = -INFINITY;
#pragma unroll
    for (int t = 0; t < MAXT; ++t) m = fmaxf(m, sv[t][e]);
    float z = 0.f;
    if (m != -INFINITY)
#pragma unroll
      for (int t = 0; t < MAXT; ++t) z += __expf(sv[t][e] - m);
    const float gm = group16_max(m);
    const float gz = group16_sum(m == -INFINITY ? 0.f : z * __expf(m - gm));
    mx[e] = gm;
    sm[e] = gz;
    if (lb.oc == 0) { sm_m[lb.wave][lb.orow + e] = gm; sm_s[lb.wave][lb.orow + e] = gz; }
  }
  __syncthreads();
  if (threadIdx.x < 16) {
    const int r = threadIdx.x, rr = lb.rb + r;
    float D = 0.f;
    if (rr < lb.rows_g) {
      float m = -INFINITY;
      for (int w = 0; w < W; ++w) m = fmaxf(m, sm_m[w][r]);
      float z = 0.f;
      for (int w = 0; w < W; ++w) z += (sm_m[w][r] == -INFINITY) ? 0.f : sm_s[w][r] * __expf(sm_m[w][r] - m);
      D = m + logf(z);
      if (nonvis_lse) {
        const int h = lb.g * sh.hg + rr / sh.T, t = rr % sh.T;
        const float nv = nonvis_lse[(static_cast<long long>(lb.p) * sh.hq + h) * sh.T + t];
        const float hi = fmaxf(D, nv), lo = fminf(D, nv);
        D = (hi == -INFINITY) ? hi : hi + log1pf(expf(lo - hi));
      }
    }
    sm_D[r] = D;
  }
  __syncthreads();
  // e = A * l_h[col], written to the grounded client rows; row sums / maxima
  float D[4], sig2[4], rsum[4], rmax[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    D[e] = sm_D[lb.orow + e];
    const float sg = sm_sig[lb.orow + e];
    sig2[e] = sg * sg;
    rsum[e] = 0.f;
    rmax[e] = 0.f;
  }
  float* E = ws.E + lb.p * ws.s_E;
#pragma unroll
  for (int t = 0; t < MAXT; ++t) {
    const int ct = lb.wave + t * W, col = ct * 16 + lb.oc;
    if (ct >= ntile || col >= sh.N) continue;
    float v[4];
    if constexpr (VEC) {
      const float nrm = sqrtf(lv[t][0] + sig2[0]);   // atom norm l_h[col], shared by the four rows
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = __expf(sv[t][e] - D[e]) * nrm;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = __expf(sv[t][e] - D[e]) * sqrtf(lv[t][e] + sig2[e]);
    }
    if constexpr (VEC) {
      *reinterpret_cast<float4*>(E + static_cast<long long>(col) * sh.ldM + mrow[0]) = make_float4(v[0], v[1], v[2], v[3]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        rsum[e] += v[e];
        rmax[e] = fmaxf(rmax[e], v[e]);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (!rvalid[e]) continue;
        E[static_cast<long long>(col) * sh.ldM + mrow[e]] = v[e];
        rsum[e] += v[e];
        rmax[e] = fmaxf(rmax[e], v[e]);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float s2 = group16_sum(rsum[e]);
    const float m2 = group16_max(rmax[e]);
    if (lb.oc == 0) { sm_s[lb.wave][lb.orow + e] = s2; sm_m[lb.wave][lb.orow + e] = m2; }
  }
  __syncthreads();
  if (threadIdx.x < 16) {
    const int r = threadIdx.x;
    if (lb.rb + r < lb.rows_g) {
      float s2 = 0.f, m2 = 0.f;
      for (int w = 0; w < W; ++w) { s2 += sm_s[w][r]; m2 = fmaxf(m2, sm_m[w][r]); }
      const long long mi = lb.mrow(sh, r);
      ws.rowsum[lb.p * ws.s_m + mi] = s2;
      ws.peak[lb.p * ws.s_m + mi] = m2;   // max_i e; scaled by the row weight later
    }
  }
}

// ---------------------------------------------------------------------------
// Head-pattern Gram (Eq. cond-head-pattern)
//   Gamma_hg = sum_(t,i) A_h A_g <w_h[i], w_g[i]>
//            = sum_i W_i[h][g] * G_i[h][g],  G_i = X_i X_i^T,
// with X_i[h][t] = e_(h,t,i) (the token's grounded atoms, one contiguous
// slice of its client row) and W_i[h][g] = <w_h[i], w_g[i]> / (l_h[i] l_g[i]).
// One wave per token at a time: X_i is staged in LDS in 64-column chunks
// (heads padded to 32), G_i accumulates on fp32 MFMA (16x16x4 tiles (0,0),
// (0,1), (1,1); the Gram is symmetric), W_i is applied in the epilogue and the
// weighted tiles accumulate over the wave's tokens.  The diagonal gives
// e2[h][i] = sum_t nu_t e_(h,t,i)^2 = nu G_hh + (nu_T - nu) X_i[h][T-1]^2.
// The block's four waves are summed in wave order into one partial per pair.
// ---------------------------------------------------------------------------
constexpr int kGramTC = 64;                 // t columns per LDS chunk
constexpr int kGramPitch = kGramTC + 4;     // floats per staged head row
constexpr int kGramTok = 2;                 // tokens per wave (kHeadTok per block)
static_assert(kGramTok * 4 == kHeadTok, "one block covers kHeadTok tokens");

template <int R>
__global__ void __launch_bounds__(256) headgram_kernel(Shape sh, Params pr, Ws ws, int write_e2) {
  constexpr int U = R + 1;                     // [Z_h[i]; sigma_h] / l_h[i]
  __shared__ __attribute__((aligned(16))) float xs[4][32 * kGramPitch];
  __shared__ float us[4][32 * U];
  const int p = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int H = sh.hq, T = sh.T;
  const int fr = lane & 15, fk = lane >> 4;
  const float nu_o = 1.f / (T - 1 + pr.terminal_q_weight);
  const float nu_last = pr.terminal_q_weight * nu_o;
  float* X = xs[wave];
  float* Uv = us[wave];
  const float* E = ws.E + p * ws.s_E;
  const float* sig = ws.sig + p * ws.s_sig;
  const float* zp = ws.z + p * ws.s_z;
  const float* qp = ws.ell + p * ws.s_ell;     // ||Z_h[i]||^2
  float* e2 = ws.e2 + p * ws.s_e2;
  floatx4 acc[3];
#pragma unroll
  for (int tl = 0; tl < 3; ++tl) acc[tl] = floatx4{0.f, 0.f, 0.f, 0.f};
  // lane h < 32 owns head h's normalised vector; the first chunk of the next
  // token and its vector load while the current token is computed
  const int hl = min(lane, H - 1);
  const float sg = sig[hl];
  float vx[32], uz[R], uq;
  auto load_token = [&](int i, int t0) {
    const float* row = E + static_cast<long long>(min(i, sh.N - 1)) * sh.ldM;
    const int tc = min(kGramTC, T - t0);
#pragma unroll
    for (int k = 0; k < 8; ++k)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int h = min(k * 4 + fk, H - 1), c = min(fr * 4 + q, tc - 1);
        vx[k * 4 + q] = row[h * T + t0 + c];
      }
  };
  auto load_vec = [&](int i) {
    const int ic = min(i, sh.N - 1);
#pragma unroll
    for (int c = 0; c < R; ++c) uz[c] = zp[static_cast<long long>(ic) * sh.hr + hl * R + c];
    uq = qp[static_cast<long long>(hl) * sh.N + ic];
  };
  auto store_chunk = [&](int tc) {
#pragma unroll
    for (int k = 0; k < 8; ++k)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int h = k * 4 + fk, c = fr * 4 + q;
        X[h * kGramPitch + c] = (h < H && c < tc) ? vx[k * 4 + q] : 0.f;
      }
  };
  auto store_vec = [&]() {
    if (lane < 32) {
      const bool ok = lane < H;
      const float inv_l = ok ? rsqrtf(uq + sg * sg) : 0.f;     // 1 / l_h[i]
#pragma unroll
      for (int c = 0; c < R; ++c) Uv[lane * U + c] = uz[c] * inv_l;
      Uv[lane * U + R] = sg * inv_l;
    }
  };
  const int tok0 = blockIdx.x * kHeadTok + wave * kGramTok;
  load_token(tok0, 0);
  load_vec(tok0);
  for (int j = 0; j < kGramTok; ++j) {
    const int i = tok0 + j;
    if (i >= sh.N) break;                                          // wave-uniform
    __builtin_amdgcn_wave_barrier();
    store_vec();
    floatx4 g[3];
#pragma unroll
    for (int tl = 0; tl < 3; ++tl) g[tl] = floatx4{0.f, 0.f, 0.f, 0.f};
    int t0 = 0;
    for (; t0 < T; t0 += kGramTC) {
      const int tc = min(kGramTC, T - t0);
      __builtin_amdgcn_wave_barrier();
      if (t0 > 0) load_token(i, t0);                               // later chunks of a long T
      store_chunk(tc);
      __builtin_amdgcn_wave_barrier();
      const int nk = (tc + 3) / 4;
      for (int kk = 0; kk < nk; ++kk) {
        const float a0 = X[fr * kGramPitch + 4 * kk + fk];
        const float a1 = X[(16 + fr) * kGramPitch + 4 * kk + fk];
        g[0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0, a0, g[0], 0, 0, 0);
        g[1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0, a1, g[1], 0, 0, 0);
        g[2] = __builtin_amdgcn_mfma_f32_16x16x4f32(a1, a1, g[2], 0, 0, 0);
      }
    }
    const int tl_last = (T - 1) - (t0 - kGramTC);   // column of t = T-1 in the last chunk
    if (j + 1 < kGramTok) {                          // next token's loads overlap the epilogue
      load_token(i + 1, 0);
      load_vec(i + 1);
    }
    __builtin_amdgcn_wave_barrier();
    // epilogue: lane holds G[16 hb + 4 fk + e][16 gb + fr]; weight
    // W[h][g] = u_h . u_g with u = [Z; sigma] / l
#pragma unroll
    for (int tl = 0; tl < 3; ++tl) {
      const int hb = tl == 2 ? 1 : 0, gb = tl == 0 ? 0 : 1;
      const int gg = 16 * gb + fr;
      float ug[U];
#pragma unroll
      for (int c = 0; c < U; ++c) ug[c] = Uv[gg * U + c];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int hh = 16 * hb + 4 * fk + e;
        float w = 0.f;
#pragma unroll
        for (int c = 0; c < U; ++c) w += Uv[hh * U + c] * ug[c];
        acc[tl][e] += g[tl][e] * w;
        if (write_e2 && tl != 1 && hh == gg && hh < H) {
          const float xl = X[hh * kGramPitch + tl_last];
          e2[static_cast<long long>(hh) * sh.N + i] = nu_o * g[tl][e] + (nu_last - nu_o) * xl * xl;
        }
      }
    }
  }
  // the block's partial: waves summed in order, one value per pair h <= g
  __syncthreads();
  float* red = &xs[0][0];   // 4 waves x 768 floats, staging buffers are free now
#pragma unroll
  for (int tl = 0; tl < 3; ++tl)
#pragma unroll
    for (int e = 0; e < 4; ++e) red[wave * 768 + tl * 256 + e * 64 + lane] = acc[tl][e];
  __syncthreads();
  // block-major partials, pairs padded to a multiple of four
  const long long npp = (sh.npairs + 3) & ~3;
  float* gp = ws.gpart + p * ws.s_gpart + blockIdx.x * npp;
  for (int x = tid; x < 768; x += 256) {
    const int tl = x / 256, e = (x / 64) % 4, l = x % 64;
    const int hb = tl == 2 ? 1 : 0, gb = tl == 0 ? 0 : 1;
    const int hh = 16 * hb + 4 * (l >> 4) + e, gg = 16 * gb + (l & 15);
    if (hh <= gg && gg < H) {
      const float v = ((red[x] + red[768 + x]) + red[2 * 768 + x]) + red[3 * 768 + x];
      gp[hh * H - hh * (hh - 1) / 2 + (gg - hh)] = v;
    }
  }
}

// ---------------------------------------------------------------------------
// Head clustering, head weights and grounded row weights.  One block per
// problem: Gamma is reduced from the per-block partials in block order
// (many loads in flight per thread), then one wave runs farthest-first with
// lane h owning head h: wave-wide max / min (DPP scans), the lowest lane
// holding the best value by ballot.
// ---------------------------------------------------------------------------

// Raised by the side stream once every bank kernel of the call has finished.
__global__ void bank_signal_kernel(int* flag) {
  if (threadIdx.x == 0) __hip_atomic_store(flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// One block per problem (occupancy is irrelevant, so the register budget goes
// to loads in flight).  Every load goes out first and coalesced: the Gram
// partials as float4 quads of pairs over groups of blocks, the grounded row
// sums as float4 runs of queries, the first pass of the row weights; partial
// sums are combined through LDS in a fixed order.
constexpr int kClusterThreads = 512;
constexpr int kClusterGB = 16;   // block partial quads in flight per thread (more spills to scratch)

__global__ void __launch_bounds__(kClusterThreads) __attribute__((amdgpu_waves_per_eu(1, 2)))
cluster_kernel(Shape sh, Params pr, Ws ws, float* trace_omega, const int* bank_flag) {
  constexpr int NT = kClusterThreads, kRW = 4;
  __shared__ float gam[kMaxHeads][kMaxHeads + 1];    // pattern Gram over the views
  __shared__ float cosm[kMaxHeads][kMaxHeads + 1];   // one view's Gamma, then the cosines
  __shared__ float4 gq[NT];
  __shared__ float hs[4 * NT];
  __shared__ float om[kMaxHeads], ab[kMaxHeads];
  __shared__ int asg[kMaxHeads];
  const int p = blockIdx.x, tid = threadIdx.x, H = sh.hq, T = sh.T, M1 = sh.mg1;
  const float* rowsum = ws.rowsum + p * ws.s_m;
  const int nb = sh.n_head_blk, npp = (sh.npairs + 3) & ~3, nq = npp / 4;
  // Gamma of a view: thread (quad qq of pairs, block group bg) adds its
  // groups' quads in block order; the groups are added in order below.  The
  // first batch of quads goes out before the row-sum loads, and every load
  // of the first batch before the first add.
  const int ngrp = max(1, NT / nq);
  const int qq = tid % nq, bg = tid / nq;
  const int bper = (nb + ngrp - 1) / ngrp;
  const int b_beg = bg * bper, b_end = min(nb, b_beg + bper);
  const bool gthr = bg < ngrp && b_beg < b_end;
  // grounded row sums in runs of four queries of one head (T a multiple of 4
  // and at most 4 NT runs per view; otherwise each head's lane adds its rows)
  const bool runs = (T & 3) == 0 && M1 <= 16 * NT;
  float zv0[kRW], pv0[kRW];
  for (int v = 0; v < sh.nviews; ++v) {
    const float* gp = ws.gpart + p * ws.s_gpart + v * ws.s_gpart1;
    const float* rs = rowsum + v * M1;
    float4 vq[kClusterGB];
    if (gthr) {
#pragma unroll
      for (int j = 0; j < kClusterGB; ++j)
        vq[j] = *reinterpret_cast<const float4*>(gp + static_cast<long long>(min(b_beg + j, b_end - 1)) * npp + 4 * qq);
    }
    if (v == 0) {
      // the first pass of the grounded row weights
#pragma unroll
      for (int k = 0; k < kRW; ++k) {
        const int m = min(k * NT + tid, sh.mg - 1);
        zv0[k] = rowsum[m];
        pv0[k] = ws.peak[p * ws.s_m + m];
      }
    }
    float4 rq[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int x = k * NT + tid;
      rq[k] = (runs && 4 * x < M1) ? *reinterpret_cast<const float4*>(rs + 4 * x) : float4{0.f, 0.f, 0.f, 0.f};
    }
    __builtin_amdgcn_sched_barrier(0);
    float4 gs = {0.f, 0.f, 0.f, 0.f};
    if (gthr) {
#pragma unroll
      for (int j = 0; j < kClusterGB; ++j)
        if (b_beg + j < b_end) { gs.x += vq[j].x; gs.y += vq[j].y; gs.z += vq[j].z; gs.w += vq[j].w; }
      for (int b0 = b_beg + kClusterGB; b0 < b_end; b0 += kClusterGB) {
#pragma unroll
        for (int j = 0; j < kClusterGB; ++j)
          vq[j] = *reinterpret_cast<const float4*>(gp + static_cast<long long>(min(b0 + j, b_end - 1)) * npp + 4 * qq);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < kClusterGB; ++j)
          if (b0 + j < b_end) { gs.x += vq[j].x; gs.y += vq[j].y; gs.z += vq[j].z; gs.w += vq[j].w; }
      }
    }
    __syncthreads();   // gq, hs, cosm and ab of the previous view are consumed
    gq[tid] = gs;
#pragma unroll
    for (int k = 0; k < 4; ++k) hs[k * NT + tid] = (rq[k].x + rq[k].y) + (rq[k].z + rq[k].w);
    __syncthreads();
    for (int hg = tid; hg < kMaxHeads * kMaxHeads; hg += NT) {
      const int h = hg / kMaxHeads, g = hg % kMaxHeads;
      if (h <= g && g < H) {
        const int x = h * H - h * (h - 1) / 2 + (g - h);   // pair (h, g) in row-major upper order
        const int q4 = x >> 2, c = x & 3;
        const float* gqf = reinterpret_cast<const float*>(gq);
        float sv = 0.f;
        for (int g2 = 0; g2 < ngrp; ++g2) sv += gqf[4 * (g2 * nq + q4) + c];
        cosm[h][g] = sv;
        cosm[g][h] = sv;
      }
    }
    if (tid < 64) {
      // mean atom norm abar_h = sum_t Z_(h,t) / (T N) of this view
      const int h = min(tid, H - 1);
      float abar = 0.f;
      if (runs) {
        for (int x = h * (T / 4); x < (h + 1) * (T / 4); ++x) abar += hs[x];
      } else {
        for (int t = 0; t < T; ++t) abar += rs[h * T + t];
      }
      if (tid < H) ab[tid] = abar / (static_cast<float>(T) * sh.N);
    }
    __syncthreads();
    // the view's share of the pattern Gram: beta_v Gamma_hg / (abar_h abar_g)
    // (the patterns are its atoms scaled to unit average norm, times
    // sqrt(beta_v)); a head without energy in the view adds nothing
    const float beta = pr.beta_view[v];
    for (int x = tid; x < H * H; x += NT) {
      const int h = x / H, g = x % H;
      const float ih = ab[h] > 0.f ? 1.f / ab[h] : 0.f, ig = ab[g] > 0.f ? 1.f / ab[g] : 0.f;
      const float c = beta * cosm[h][g] * ih * ig;
      gam[h][g] = v == 0 ? c : gam[h][g] + c;
    }
  }
  __syncthreads();
  // cosines of the head patterns, all threads
  for (int x = tid; x < H * H; x += NT) {
    const int h = x / H, g = x % H;
    const float hh = gam[h][h], gg = gam[g][g];
    cosm[h][g] = gam[h][g] / ((hh > 0.f ? sqrtf(hh) : 1.f) * (gg > 0.f ? sqrtf(gg) : 1.f));
  }
  __syncthreads();
  if (tid < 64) {
    const int lane = tid, h = lane;
    const bool valid = h < H;
    const float ghh = valid ? gam[h][h] : 0.f;
    const bool active = valid && ghh > 0.f;
    const int n_active = __popcll(__ballot(active));
    float w_h = 0.f;
    int cl = -1;
    if (n_active > 0) {
      // first centre: the largest pre-normalisation pattern (its squared norm
      // is the pattern Gram's diagonal)
      const float v = active ? sqrtf(ghh) : -INFINITY;
      const float vbest = wave_max(v);
      const int idx = __ffsll(static_cast<unsigned long long>(__ballot(active && v == vbest))) - 1;
      int nc = 1;
      bool is_c = h == idx;
      float maxcos = valid ? cosm[h][idx] : -INFINITY;
      // each head's nearest centre so far (ties to the earlier centre)
      float bv = maxcos;
      int best = 0;
      const int want = min(pr.max_head_clusters, n_active);
      while (nc < want) {
        // next centre: the active non-centre head least similar to every centre
        const bool cand = active && !is_c;
        const float cv = cand ? maxcos : INFINITY;
        const float cbest = wave_min(cv);
        const unsigned long long cm = static_cast<unsigned long long>(__ballot(cand && cv == cbest));
        if (cm == 0ull) break;
        const int ci = __ffsll(cm) - 1;
        const float cc = valid ? cosm[h][ci] : -INFINITY;
        if (cc > bv) { bv = cc; best = nc; }
        ++nc;
        is_c |= h == ci;
        maxcos = fmaxf(maxcos, cc);
      }
      if (active) cl = best;
      if (valid) asg[h] = cl;
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
      // clusters, dispersion d_h = 1 - u_h . mu_c and inverse-dispersion weights
      int n_clusters = 0;
      for (int c = 0; c < nc; ++c) n_clusters += __ballot(cl == c) != 0ull;
      // members of the head's cluster (adding zeros for the others leaves
      // the sum unchanged)
      float s_h = 0.f;
#pragma unroll
      for (int g = 0; g < kMaxHeads; ++g) s_h += (g < H && asg[g] == cl) ? cosm[h][g] : 0.f;
      if (cl < 0) s_h = 0.f;
      float inv = 0.f;
      for (int c = 0; c < nc; ++c) {
        const float tot = wave_sum(cl == c ? s_h : 0.f);
        if (cl == c) {
          const float disp = 1.f - s_h / sqrtf(fmaxf(tot, 0.f));
          inv = 1.f / (disp + pr.disp_eps);
        }
      }
      for (int c = 0; c < nc; ++c) {
        const float isum = wave_sum(cl == c ? inv : 0.f);
        if (cl == c) w_h = inv / isum / static_cast<float>(n_clusters);
      }
    }
    if (valid) {
      om[h] = w_h;
      ws.omega[p * ws.s_om + h] = w_h;
      if (trace_omega) trace_omega[static_cast<long long>(p) * H + h] = w_h;
    }
  }
  __syncthreads();
  // grounded row weights beta_v omega_h nu_t a_(h,t) / Z_(h,t) of every view
  const float nu_o = 1.f / (T - 1 + pr.terminal_q_weight);
  for (int m0 = 0; m0 < sh.mg; m0 += NT * kRW) {
    float zv[kRW], pv[kRW];
#pragma unroll
    for (int k = 0; k < kRW; ++k) {
      if (m0 == 0) {
        zv[k] = zv0[k];
        pv[k] = pv0[k];
      } else {
        const int m = min(m0 + k * NT + tid, sh.mg - 1);
        zv[k] = rowsum[m];
        pv[k] = ws.peak[p * ws.s_m + m];
      }
    }
#pragma unroll
    for (int k = 0; k < kRW; ++k) {
      const int m = m0 + k * NT + tid;
      if (m < sh.mg) {
        const int v = m / M1, mm = m - v * M1, h = mm / T, t = mm % T;
        const float nu = (t == T - 1) ? pr.terminal_q_weight * nu_o : nu_o;
        const float a = (zv[k] > 0.f) ? pr.beta_view[v] * om[h] * nu / zv[k] : 0.f;
        ws.alpha[p * ws.s_m + m] = a;
        ws.peak[p * ws.s_m + m] = pv[k] * a;
      }
    }
  }
  // the bank kernels run on another stream; the kernel after this one reads
  // their client rows, so this one ends only once the side stream has raised
  // bank_flag (one thread per block waits; every wait is bounded)
  if (bank_flag && tid == 0) {
    const unsigned long long t0 = static_cast<unsigned long long>(wall_clock64());
    for (int spin = 0; __hip_atomic_load(bank_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 1; ++spin) {
      if ((spin & 255) == 255 && static_cast<unsigned long long>(wall_clock64()) - t0 > kJoinWaitTicks) {
        raise_status(ws.cnt + p * ws.s_cnt, kStatusBank);
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
  }
}

// Empty grounded bank (T = 0): omega = 0 and uniform energy ebar = 1.
__global__ void no_grounded_kernel(Shape sh, Ws ws, float* trace_omega) {
  const int p = blockIdx.y;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < sh.N; i += gridDim.x * blockDim.x)
    ws.ebar[p * ws.s_eb + i] = 1.f;
  if (blockIdx.x == 0) {
    for (int h = threadIdx.x; h < sh.hq; h += blockDim.x) {
      ws.omega[p * ws.s_om + h] = 0.f;
      if (trace_omega) trace_omega[static_cast<long long>(p) * sh.hq + h] = 0.f;
    }
  }
}

// ---------------------------------------------------------------------------
// host launchers
// ---------------------------------------------------------------------------
// Row norms of a historical view's states into ws.n2h (no per-call reset).
template <typename T>
static void launch_view_rownorm(const Shape& sh, const Ws& ws, const void* hidden, hipStream_t st) {
  Ws wv = ws;
  wv.n2 = ws.n2h;
  wv.s_n = ws.s_n2h;
  hipLaunchKernelGGL(rownorm_kernel<T>, dim3((sh.N + 3) / 4, sh.B), dim3(256), 0, st, sh, wv,
                     static_cast<const T*>(hidden), 0, 0);
}

// One message view: value probe and mass coordinate from the view's states
// and folded probe, the native slice into the view's grounded rows, and the
// view's head-pattern Gram partials (the current view also leaves the
// energy numerators).  `sv` counts one view's grounded rows; `wv` points at
// the view's rows, norms and Gram partials.
template <typename T>
static hipError_t message_view(const Shape& sv, const Params& pr, const Ws& wv, const MsgView& mv, bool current,
                               hipStream_t st) {
  const T* hidden = static_cast<const T*>(mv.hidden);
  Params pv = pr;
  pv.probe_bias = mv.probe_bias;
  timer_mark(kStProbe, true, st);
  RowOperand<T> A{hidden, sv.d, static_cast<long long>(sv.N) * sv.d, nullptr, 0, sv.N};
  RowOperand<T> Bp{static_cast<const T*>(mv.probe), sv.d, 0, nullptr, 0, sv.hr};
  // split the d-long contraction so four times as many blocks stream hidden
  const int ksplit = (sv.d % (64 * kProbeSplit) == 0) ? kProbeSplit : 1;
  ProbeSplitEpi pe{wv, sv.hr, static_cast<long long>(sv.N) * sv.hr};
  hipError_t err = launch_gemm_nt<T, 64, 64>(A, Bp, sv.d, sv.B, pe, st, ksplit);
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(sigma_ell_kernel, dim3((sv.N + 63) / 64, (sv.hq + 3) / 4, sv.B), dim3(256), 0, st, sv, pv, wv,
                     ksplit);
  timer_mark(kStProbe, false, st);
  const dim3 lg((sv.hg * sv.T + 15) / 16 * sv.lsplit, sv.hkv, sv.B);
  const dim3 lr((sv.hg * sv.T + 15) / 16, sv.hkv, sv.B);
  // every tile of a block's rows fits the registers of its eight waves
  const bool staged_ok = std::is_same<T, bf16_t>::value && (sv.T & 15) == 0 && sv.dh <= 128;
  // the register kernel (one pass, keys read once) while its 16-row blocks
  // number at most one per CU; many images fill the chip better with the
  // staged column-range kernels
  const bool reg = (sv.N + 15) / 16 <= 8 * kLogitRegTiles &&
                   (!staged_ok || static_cast<long long>(lr.x) * lr.y * lr.z <= 256);
  const T* q = static_cast<const T*>(mv.text_q);
  const T* k = static_cast<const T*>(mv.vis_k);
  const float* nonvis_lse = mv.nonvis_lse;
  timer_mark(kStLogits, true, st);
  bool wide = false;
  if constexpr (std::is_same<T, bf16_t>::value) {
    if (!reg && staged_ok) {
      wide = true;
      // staged blocks of 16 kStW rows: split the columns until about four
      // blocks per CU, keeping at least two stages per range
      Shape sw = sv;
      const int row_blocks = (sv.hg * sv.T + kStRows - 1) / kStRows;
      const long long rbw = static_cast<long long>(row_blocks) * sv.hkv * sv.B;
      const long long ntile = (sv.N + 15) / 16;
      long long ls = (1024 + rbw - 1) / rbw;
      ls = std::min<long long>(ls, ntile / (2 * kStSG));
      sw.lsplit = static_cast<int>(std::max<long long>(1, std::min<long long>(ls, kLogitSplit)));
      const dim3 gw(static_cast<unsigned>(row_blocks * sw.lsplit), sv.hkv, sv.B);
      switch (sv.dh) {
#define GMC_STAGE(DH)                                                                                        \
        case DH:                                                                                             \
          hipLaunchKernelGGL(logits_lse_stage_kernel<DH>, gw, dim3(64 * kStW), 0, st, sw, pv, wv, q, k);     \
          hipLaunchKernelGGL(logits_stage_kernel<DH>, gw, dim3(64 * kStW), 0, st, sw, wv, q, k, nonvis_lse);  \
          break;
        GMC_STAGE(32) GMC_STAGE(64) GMC_STAGE(96) GMC_STAGE(128)
#undef GMC_STAGE
        default: return hipErrorInvalidValue;
      }
    }
  }
  if (!wide) switch (sv.dh) {
#define GMC_LOGITS(DH)                                                                                         \
    case DH:                                                                                                   \
      if constexpr (logit_reg_ok<T, DH>()) {                                                                  \
        if (reg) {                                                                                             \
          if ((sv.T & 15) == 0)                                                                                \
            hipLaunchKernelGGL((logits_reg_kernel<T, DH, kLogitRegTiles, true>), lr, dim3(512), 0, st, sv, pv, wv, q, \
                               k, nonvis_lse);                                                                 \
          else                                                                                                 \
            hipLaunchKernelGGL((logits_reg_kernel<T, DH, kLogitRegTiles, false>), lr, dim3(512), 0, st, sv, pv, wv, \
                               q, k, nonvis_lse);                                                              \
          break;                                                                                               \
        }                                                                                                      \
      }                                                                                                        \
      hipLaunchKernelGGL((logits_lse_kernel<T, DH>), lg, dim3(64 * logit_waves<T, DH>()), 0, st, sv, pv, wv, q, k); \
      hipLaunchKernelGGL((logits_kernel<T, DH>), lg, dim3(64 * logit_waves<T, DH>()), 0, st, sv, wv, q, k,       \
                         nonvis_lse);                                                                          \
      break;
    GMC_LOGITS(32) GMC_LOGITS(64) GMC_LOGITS(96) GMC_LOGITS(128)
    GMC_LOGITS(160) GMC_LOGITS(192) GMC_LOGITS(224) GMC_LOGITS(256)
#undef GMC_LOGITS
    default: return hipErrorInvalidValue;
  }
  timer_mark(kStLogits, false, st);
  timer_mark(kStHeads, true, st);
  const int we2 = current ? 1 : 0;
  switch (sv.r) {
#define GMC_HEADGRAM(R) \
    case R: hipLaunchKernelGGL(headgram_kernel<R>, dim3(sv.n_head_blk, sv.B), dim3(256), 0, st, sv, pv, wv, we2); break;
    GMC_HEADGRAM(1) GMC_HEADGRAM(2) GMC_HEADGRAM(3) GMC_HEADGRAM(4)
    GMC_HEADGRAM(5) GMC_HEADGRAM(6) GMC_HEADGRAM(7) GMC_HEADGRAM(8)
#undef GMC_HEADGRAM
    default: return hipErrorInvalidValue;
  }
  timer_mark(kStHeads, false, st);
  return hipGetLastError();
}

template <typename T>
static hipError_t message_impl(const Shape& sh, const Params& pr, const Ws& ws, const MsgView* views,
                               float* trace_omega, const int* bank_flag, hipStream_t st) {
  if (sh.T == 0) {
    // no grounded rows: the value probe is not needed either
    timer_mark(kStHeads, true, st);
    hipLaunchKernelGGL(no_grounded_kernel, dim3((sh.N + 255) / 256, sh.B), dim3(256), 0, st, sh, ws,
                       trace_omega);
    timer_mark(kStHeads, false, st);
    return hipGetLastError();
  }
  Shape sv = sh;
  sv.mg = sh.mg1;
  for (int v = 0; v < sh.nviews; ++v) {
    Ws wv = ws;
    wv.E = ws.E + static_cast<long long>(v) * sh.mg1;
    wv.rowsum = ws.rowsum + static_cast<long long>(v) * sh.mg1;
    wv.peak = ws.peak + static_cast<long long>(v) * sh.mg1;
    wv.gpart = ws.gpart + v * ws.s_gpart1;
    if (v > 0) {
      launch_view_rownorm<T>(sh, ws, views[v].hidden, st);
      wv.n2 = ws.n2h;
      wv.s_n = ws.s_n2h;
    }
    const hipError_t err = message_view<T>(sv, pr, wv, views[v], v == 0, st);
    if (err != hipSuccess) return err;
  }
  timer_mark(kStHeads, true, st);
  hipLaunchKernelGGL(cluster_kernel, dim3(sh.B), dim3(kClusterThreads), 0, st, sh, pr, ws, trace_omega, bank_flag);
  timer_mark(kStHeads, false, st);
  return hipGetLastError();
}

hipError_t launch_rownorm(const Shape& sh, const Ws& ws, const void* hidden, int call_tag, hipStream_t st) {
  timer_mark(kStInit, true, st);
  if (sh.dtype == 0)
    hipLaunchKernelGGL(rownorm_kernel<float>, dim3((sh.N + 3) / 4, sh.B), dim3(256), 0, st, sh, ws,
                       static_cast<const float*>(hidden), call_tag, 1);
  else
    hipLaunchKernelGGL(rownorm_kernel<bf16_t>, dim3((sh.N + 3) / 4, sh.B), dim3(256), 0, st, sh, ws,
                       static_cast<const bf16_t*>(hidden), call_tag, 1);
  timer_mark(kStInit, false, st);
  return hipGetLastError();
}

hipError_t launch_bank_gate(const Shape& sh, const Ws& ws, int call_tag, hipStream_t st) {
  hipLaunchKernelGGL(bank_gate_kernel, dim3(1), dim3(256), 0, st, sh, ws, call_tag);
  return hipGetLastError();
}

hipError_t launch_message(const Shape& sh, const Params& pr, const Ws& ws, const MsgView* views,
                          float* trace_omega, const int* bank_flag, hipStream_t st) {
  if (sh.dtype == 0) return message_impl<float>(sh, pr, ws, views, trace_omega, bank_flag, st);
  return message_impl<bf16_t>(sh, pr, ws, views, trace_omega, bank_flag, st);
}

hipError_t launch_bank_signal(int* flag, hipStream_t st) {
  hipLaunchKernelGGL(bank_signal_kernel, dim3(1), dim3(64), 0, st, flag);
  return hipGetLastError();
}

}  // namespace gmc
