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
// Squared row norms of the hidden states: one wave per token.
// ---------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256) rownorm_kernel(Shape sh, Ws ws, const T* hidden) {
  const int p = blockIdx.y;
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (i >= sh.N) return;
  const T* row = hidden + (static_cast<long long>(p) * sh.N + i) * sh.d;
  float s = 0.f;
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
  if (lane == 0) ws.n2[p * ws.s_n + i] = s;
}

// Probe GEMM epilogue: Z[i][c] = (h_i . G_c) / sqrt(mean h_i^2 + eps), the
// folded value path applied to the next block's RMSNorm of h_i.
struct ProbeEpi {
  Ws ws;
  int d;
  float rms_eps;
  static constexpr bool kRowStats = false;
  int hr;
  __device__ void store(int p, int r, int c, float acc) const {
    const float ms = ws.n2[p * ws.s_n + r] / static_cast<float>(d);
    ws.z[p * ws.s_z + static_cast<long long>(r) * hr + c] = acc * rsqrtf(ms + rms_eps);
  }
  __device__ float value(int, int, int, float) const { return 0.f; }
  __device__ void row_stats(int, int, int, float, float) const {}
};

// sigma_h = sqrt(lambda) max(||Z_h||_F / sqrt(N r), eps) and
// l_h[i] = ||[Z_h[i]; sigma_h]||.  One block per (head, problem).
__global__ void __launch_bounds__(256) sigma_ell_kernel(Shape sh, Params pr, Ws ws) {
  __shared__ float red[16];
  const int h = blockIdx.x, p = blockIdx.y;
  const float* z = ws.z + p * ws.s_z;
  float acc = 0.f;
  for (int i = threadIdx.x; i < sh.N; i += blockDim.x) {
    const float* zi = z + static_cast<long long>(i) * sh.hr + h * sh.r;
    float s = 0.f;
    for (int c = 0; c < sh.r; ++c) s += zi[c] * zi[c];
    acc += s;
  }
  const float fro2 = block_sum(acc, red);
  const float mean2 = fro2 / (static_cast<float>(sh.N) * sh.r);
  const float sig = sqrtf(pr.lambda_mass) * fmaxf(sqrtf(mean2), pr.eps_mass);
  if (threadIdx.x == 0) ws.sig[p * ws.s_sig + h] = sig;
  float* ell = ws.ell + p * ws.s_ell + static_cast<long long>(h) * sh.N;
  for (int i = threadIdx.x; i < sh.N; i += blockDim.x) {
    const float* zi = z + static_cast<long long>(i) * sh.hr + h * sh.r;
    float s = 0.f;
    for (int c = 0; c < sh.r; ++c) s += zi[c] * zi[c];
    ell[i] = sqrtf(s + sig * sig);
  }
}

// ---------------------------------------------------------------------------
// Native message slice and grounded energies.
// Block = 16 rows (h,t) of one kv group x all N visual columns; the 4 waves
// split the 16-column tiles.  Pass 1: online max / sum-exp of the logits
// q.k/sqrt(dh).  Pass 2: recompute the logits (cheaper than storing them),
// e = exp(s - D) * l_h[i] with D the (optionally nonvisual-extended)
// log-sum-exp, write e to the grounded client rows, and reduce row sums and
// row maxima.  Nothing but e ever reaches HBM.
// ---------------------------------------------------------------------------
template <typename T, int DH>
__global__ void __launch_bounds__(256)
logits_kernel(Shape sh, Ws ws, const T* text_q, const T* vis_k, const float* nonvis_lse) {
  constexpr int KS = DH / 32;
  __shared__ float sm_m[4][16], sm_s[4][16];
  __shared__ float sm_D[16];
  const int p = blockIdx.z, g = blockIdx.y;
  const int rows_g = sh.hg * sh.T;
  const int rb = blockIdx.x * 16;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int fr = lane & 15, fk = (lane >> 4) * 8;
  const float scale = rsqrtf(static_cast<float>(DH));

  // A operand: query row rb + fr of this group
  Frag<T> qf[KS];
  {
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
  }
  const T* kbase = vis_k + static_cast<long long>(p) * sh.N * sh.hkv * DH + g * DH;
  const long long kstride = static_cast<long long>(sh.hkv) * DH;
  const int ntile = (sh.N + 15) / 16;
  const int orow = (lane >> 4) * 4, oc = lane & 15;

  auto tile_logits = [&](int ct) -> floatx4 {
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
    const int col = ct * 16 + fr;
    if (col < sh.N) {
      const T* kr = kbase + col * kstride;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) acc = mma(qf[ks], frag_load<T>(kr + ks * 32 + fk), acc);
    } else {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) acc = mma(qf[ks], frag_zero<T>(), acc);
    }
    return acc;
  };

  // pass 1: online (max, sum exp) per row, lane-local over its columns
  float mx[4], sm[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) { mx[e] = -INFINITY; sm[e] = 0.f; }
  for (int ct = wave; ct < ntile; ct += 4) {
    const floatx4 acc = tile_logits(ct);
    if (ct * 16 + oc < sh.N) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float s = acc[e] * scale;
        const float nm = fmaxf(mx[e], s);
        sm[e] = sm[e] * expf(mx[e] - nm) + expf(s - nm);
        mx[e] = nm;
      }
    }
  }
  // merge across the 16 lanes of a row group, then across waves
#pragma unroll
  for (int e = 0; e < 4; ++e) {
#pragma unroll
    for (int o = 8; o > 0; o >>= 1) {
      const float om = __shfl_xor(mx[e], o, kWave), os = __shfl_xor(sm[e], o, kWave);
      const float nm = fmaxf(mx[e], om);
      sm[e] = (nm == -INFINITY) ? 0.f : sm[e] * expf(mx[e] - nm) + os * expf(om - nm);
      mx[e] = nm;
    }
    if (oc == 0) { sm_m[wave][orow + e] = mx[e]; sm_s[wave][orow + e] = sm[e]; }
  }
  __syncthreads();
  if (threadIdx.x < 16) {
    const int r = threadIdx.x;
    float m = -INFINITY;
    for (int w = 0; w < 4; ++w) m = fmaxf(m, sm_m[w][r]);
    float s = 0.f;
    for (int w = 0; w < 4; ++w) s += (sm_m[w][r] == -INFINITY) ? 0.f : sm_s[w][r] * expf(sm_m[w][r] - m);
    float D = m + logf(s);
    const int rr = rb + r;
    if (nonvis_lse && rr < rows_g) {
      const int h = g * sh.hg + rr / sh.T, t = rr % sh.T;
      const float nv = nonvis_lse[(static_cast<long long>(p) * sh.hq + h) * sh.T + t];
      const float hi = fmaxf(D, nv), lo = fminf(D, nv);
      D = (hi == -INFINITY) ? hi : hi + log1pf(expf(lo - hi));
    }
    sm_D[r] = D;
  }
  __syncthreads();

  // pass 2: write e = A * l and reduce row sums / maxima
  float D[4], rsum[4], rmax[4];
  int hrow[4];
  long long mrow[4];
  bool rvalid[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int rr = rb + orow + e;
    rvalid[e] = rr < rows_g;
    const int h = g * sh.hg + (rvalid[e] ? rr / sh.T : 0), t = rvalid[e] ? rr % sh.T : 0;
    hrow[e] = h;
    mrow[e] = static_cast<long long>(h) * sh.T + t;
    D[e] = sm_D[orow + e];
    rsum[e] = 0.f;
    rmax[e] = 0.f;
  }
  float* E = ws.E + p * ws.s_E;
  const float* ell = ws.ell + p * ws.s_ell;
  for (int ct = wave; ct < ntile; ct += 4) {
    const floatx4 acc = tile_logits(ct);
    const int col = ct * 16 + oc;
    if (col < sh.N) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (!rvalid[e]) continue;
        const float a = expf(acc[e] * scale - D[e]);
        const float v = a * ell[static_cast<long long>(hrow[e]) * sh.N + col];
        E[mrow[e] * sh.ldE + col] = v;
        rsum[e] += v;
        rmax[e] = fmaxf(rmax[e], v);
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float s = group16_sum(rsum[e]);
    const float m = group16_max(rmax[e]);
    if (oc == 0) { sm_s[wave][orow + e] = s; sm_m[wave][orow + e] = m; }
  }
  __syncthreads();
  if (threadIdx.x < 16) {
    const int r = threadIdx.x, rr = rb + r;
    if (rr < rows_g) {
      const int h = g * sh.hg + rr / sh.T, t = rr % sh.T;
      float s = 0.f, m = 0.f;
      for (int w = 0; w < 4; ++w) { s += sm_s[w][r]; m = fmaxf(m, sm_m[w][r]); }
      const long long mi = static_cast<long long>(h) * sh.T + t;
      ws.rowsum[p * ws.s_m + mi] = s;
      ws.peak[p * ws.s_m + mi] = m;   // max_i e; scaled by the row weight later
    }
  }
}

// ---------------------------------------------------------------------------
// Head-pattern Gram Gamma_hg = sum_(t,i) A_h A_g <w_h[i], w_g[i]>
//   = sum_i [<w_h,w_g>/(l_h l_g)](i) * sum_t e_h[t,i] e_g[t,i]
// and e2[h][i] = sum_t nu_t e_h[t,i]^2.  One block per 16 tokens; the t axis
// streams through LDS in chunks of 16; each thread owns (token, pair-slot).
// ---------------------------------------------------------------------------
constexpr int kTC = 16;
constexpr int kPairsPerThread = (kMaxHeads * (kMaxHeads + 1) / 2 + 15) / 16;

__global__ void __launch_bounds__(256) headgram_kernel(Shape sh, Params pr, Ws ws) {
  __shared__ float tileE[kMaxHeads * kTC * kHeadTok];
  __shared__ float zt[kHeadTok * kMaxHeads * kMaxProbe];
  __shared__ float lt[kMaxHeads * kHeadTok];
  __shared__ short pair_h[kMaxHeads * (kMaxHeads + 1) / 2], pair_g[kMaxHeads * (kMaxHeads + 1) / 2];
  const int p = blockIdx.y, i0 = blockIdx.x * kHeadTok;
  const int tid = threadIdx.x, il = tid & 15, slot = tid >> 4;
  const int H = sh.hq, T = sh.T;
  if (tid == 0) {
    int q = 0;
    for (int h = 0; h < H; ++h)
      for (int g = h; g < H; ++g) { pair_h[q] = h; pair_g[q] = g; ++q; }
  }
  const float nu_o = 1.f / (T - 1 + pr.terminal_q_weight);
  const float nu_last = pr.terminal_q_weight * nu_o;
  float acc[kPairsPerThread];
#pragma unroll
  for (int q = 0; q < kPairsPerThread; ++q) acc[q] = 0.f;
  float e2a[2] = {0.f, 0.f};
  const float* E = ws.E + p * ws.s_E;
  const int i = i0 + il;
  for (int t0 = 0; t0 < T; t0 += kTC) {
    const int tc = min(kTC, T - t0);
    __syncthreads();
    for (int x = tid; x < H * kTC * kHeadTok; x += 256) {
      const int ii = x % kHeadTok, tt = (x / kHeadTok) % kTC, h = x / (kHeadTok * kTC);
      float v = 0.f;
      if (tt < tc && i0 + ii < sh.N) v = E[(static_cast<long long>(h) * T + t0 + tt) * sh.ldE + i0 + ii];
      tileE[x] = v;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kPairsPerThread; ++q) {
      const int pq = slot + 16 * q;
      if (pq < sh.npairs) {
        const float* eh = &tileE[pair_h[pq] * kTC * kHeadTok + il];
        const float* eg = &tileE[pair_g[pq] * kTC * kHeadTok + il];
        float s = 0.f;
        for (int tt = 0; tt < tc; ++tt) s += eh[tt * kHeadTok] * eg[tt * kHeadTok];
        acc[q] += s;
      }
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int h = slot + 16 * j;
      if (h < H) {
        const float* eh = &tileE[h * kTC * kHeadTok + il];
        float s = 0.f;
        for (int tt = 0; tt < tc; ++tt) {
          const float nu = (t0 + tt == T - 1) ? nu_last : nu_o;
          s += nu * eh[tt * kHeadTok] * eh[tt * kHeadTok];
        }
        e2a[j] += s;
      }
    }
  }
  // per-token pattern weights <w_h, w_g> / (l_h l_g)
  __syncthreads();
  for (int x = tid; x < kHeadTok * sh.hr; x += 256) {
    const int ii = x / sh.hr, c = x % sh.hr;
    zt[x] = (i0 + ii < sh.N) ? ws.z[p * ws.s_z + static_cast<long long>(i0 + ii) * sh.hr + c] : 0.f;
  }
  for (int x = tid; x < H * kHeadTok; x += 256) {
    const int h = x / kHeadTok, ii = x % kHeadTok;
    lt[x] = (i0 + ii < sh.N) ? ws.ell[p * ws.s_ell + static_cast<long long>(h) * sh.N + i0 + ii] : 1.f;
  }
  __syncthreads();
  const float* sig = ws.sig + p * ws.s_sig;
  float* gp = ws.gpart + p * ws.s_gpart + static_cast<long long>(blockIdx.x) * sh.npairs;
#pragma unroll
  for (int q = 0; q < kPairsPerThread; ++q) {
    const int pq = slot + 16 * q;
    float v = 0.f;
    if (pq < sh.npairs && i < sh.N) {
      const int h = pair_h[pq], g = pair_g[pq];
      float dot = sig[h] * sig[g];
      for (int c = 0; c < sh.r; ++c) dot += zt[il * sh.hr + h * sh.r + c] * zt[il * sh.hr + g * sh.r + c];
      v = acc[q] * dot / (lt[h * kHeadTok + il] * lt[g * kHeadTok + il]);
    }
    v = group16_sum(v);
    if (il == 0 && pq < sh.npairs) gp[pq] = v;
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int h = slot + 16 * j;
    if (h < H && i < sh.N) ws.e2[p * ws.s_e2 + static_cast<long long>(h) * sh.N + i] = e2a[j];
  }
}

// ---------------------------------------------------------------------------
// Head clustering, head weights, grounded row weights and energy.
// One block per problem.  Gamma is reduced from the per-block partials in a
// fixed order; farthest-first clustering runs on one thread (Hq <= 32).
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256) cluster_kernel(Shape sh, Params pr, Ws ws, float* trace_omega,
                                                      float* trace_ebar) {
  __shared__ float gam[kMaxHeads][kMaxHeads];
  __shared__ float cosm[kMaxHeads][kMaxHeads];
  __shared__ float abar[kMaxHeads];
  __shared__ float om[kMaxHeads];
  __shared__ float red[16];
  const int p = blockIdx.x, tid = threadIdx.x, H = sh.hq, T = sh.T;
  const float* gp = ws.gpart + p * ws.s_gpart;
  for (int q = tid; q < sh.npairs; q += blockDim.x) {
    int h = 0, rem = q;
    while (rem >= H - h) { rem -= H - h; ++h; }
    const int g = h + rem;
    float s = 0.f;
    for (int b = 0; b < sh.n_head_blk; ++b) s += gp[static_cast<long long>(b) * sh.npairs + q];
    gam[h][g] = s;
    gam[g][h] = s;
  }
  const float* rowsum = ws.rowsum + p * ws.s_m;
  for (int h = tid; h < H; h += blockDim.x) {
    float s = 0.f;
    for (int t = 0; t < T; ++t) s += rowsum[h * T + t];
    abar[h] = s / (static_cast<float>(T) * sh.N);
  }
  __syncthreads();
  if (tid == 0) {
    bool active[kMaxHeads];
    int n_active = 0;
    float nrm[kMaxHeads];
    for (int h = 0; h < H; ++h) {
      active[h] = gam[h][h] > 0.f;
      n_active += active[h];
      nrm[h] = active[h] ? sqrtf(gam[h][h]) : 1.f;
      om[h] = 0.f;
    }
    for (int h = 0; h < H; ++h)
      for (int g = 0; g < H; ++g) cosm[h][g] = gam[h][g] / (nrm[h] * nrm[g]);
    if (n_active > 0) {
      int centres[kMaxHeads];
      int nc = 0;
      // first centre: largest pre-normalisation pattern sqrt(beta Gamma_hh) / abar_h
      float best = -INFINITY;
      int bi = -1;
      for (int h = 0; h < H; ++h) {
        if (!active[h]) continue;
        const float v = sqrtf(pr.beta_msg * gam[h][h]) / (abar[h] > 0.f ? abar[h] : 1.f);
        if (v > best) { best = v; bi = h; }
      }
      if (bi < 0) bi = 0;
      centres[nc++] = bi;
      const int want = min(pr.max_head_clusters, n_active);
      while (nc < want) {
        float bv = INFINITY;
        int bh = -1;
        for (int h = 0; h < H; ++h) {
          if (!active[h]) continue;
          bool is_c = false;
          for (int c = 0; c < nc; ++c) is_c |= centres[c] == h;
          if (is_c) continue;
          float v = -INFINITY;
          for (int c = 0; c < nc; ++c) v = fmaxf(v, cosm[h][centres[c]]);
          if (v < bv) { bv = v; bh = h; }
        }
        if (bh < 0) break;
        centres[nc++] = bh;
      }
      int assign[kMaxHeads];
      int count[kMaxHeads];
      for (int c = 0; c < nc; ++c) count[c] = 0;
      for (int h = 0; h < H; ++h) {
        assign[h] = -1;
        if (!active[h]) continue;
        int bc = 0;
        float bv = cosm[h][centres[0]];
        for (int c = 1; c < nc; ++c)
          if (cosm[h][centres[c]] > bv) { bv = cosm[h][centres[c]]; bc = c; }
        assign[h] = bc;
        ++count[bc];
      }
      int n_clusters = 0;
      for (int c = 0; c < nc; ++c) n_clusters += count[c] > 0;
      for (int c = 0; c < nc; ++c) {
        if (count[c] == 0) continue;
        float tot = 0.f;
        for (int h = 0; h < H; ++h)
          if (assign[h] == c)
            for (int g = 0; g < H; ++g)
              if (assign[g] == c) tot += cosm[h][g];
        const float mean_norm = sqrtf(fmaxf(tot, 0.f));
        float inv[kMaxHeads];
        float isum = 0.f;
        for (int h = 0; h < H; ++h) {
          if (assign[h] != c) continue;
          float s = 0.f;
          for (int g = 0; g < H; ++g)
            if (assign[g] == c) s += cosm[h][g];
          const float disp = 1.f - s / mean_norm;
          inv[h] = 1.f / (disp + pr.disp_eps);
          isum += inv[h];
        }
        for (int h = 0; h < H; ++h)
          if (assign[h] == c) om[h] = inv[h] / isum / static_cast<float>(n_clusters);
      }
    }
  }
  __syncthreads();
  for (int h = tid; h < H; h += blockDim.x) {
    ws.omega[p * ws.s_om + h] = om[h];
    if (trace_omega) trace_omega[static_cast<long long>(p) * H + h] = om[h];
  }
  // grounded row weights beta_msg omega_h nu_t a_(h,t) / Z_(h,t)
  const float nu_o = 1.f / (T - 1 + pr.terminal_q_weight);
  for (int m = tid; m < sh.mg; m += blockDim.x) {
    const int h = m / T, t = m % T;
    const float nu = (t == T - 1) ? pr.terminal_q_weight * nu_o : nu_o;
    const float z = rowsum[m];
    const float a = (z > 0.f) ? pr.beta_msg * om[h] * nu / z : 0.f;
    ws.alpha[p * ws.s_m + m] = a;
    ws.peak[p * ws.s_m + m] *= a;
  }
  // e_i = sqrt(sum_h omega_h sum_t nu_t e^2); ebar = e / mean(e), fallback 1
  const float* e2 = ws.e2 + p * ws.s_e2;
  float local = 0.f;
  for (int i = tid; i < sh.N; i += blockDim.x) {
    float s = 0.f;
    for (int h = 0; h < H; ++h) s += om[h] * e2[static_cast<long long>(h) * sh.N + i];
    local += sqrtf(s);
  }
  const float mean = block_sum(local, red) / static_cast<float>(sh.N);
  float* eb = ws.ebar + p * ws.s_eb;
  for (int i = tid; i < sh.N; i += blockDim.x) {
    float v = 1.f;
    if (mean > 0.f) {
      float s = 0.f;
      for (int h = 0; h < H; ++h) s += om[h] * e2[static_cast<long long>(h) * sh.N + i];
      v = sqrtf(s) / mean;
    }
    eb[i] = v;
    if (trace_ebar) trace_ebar[static_cast<long long>(p) * sh.N + i] = v;
  }
}

// Empty grounded bank (T = 0): omega = 0, ebar = 1.
__global__ void no_grounded_kernel(Shape sh, Ws ws, float* trace_omega, float* trace_ebar) {
  const int p = blockIdx.y;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < sh.N; i += gridDim.x * blockDim.x) {
    ws.ebar[p * ws.s_eb + i] = 1.f;
    if (trace_ebar) trace_ebar[static_cast<long long>(p) * sh.N + i] = 1.f;
  }
  if (blockIdx.x == 0)
    for (int h = threadIdx.x; h < sh.hq; h += blockDim.x) {
      ws.omega[p * ws.s_om + h] = 0.f;
      if (trace_omega) trace_omega[static_cast<long long>(p) * sh.hq + h] = 0.f;
    }
}

// ---------------------------------------------------------------------------
// host launchers
// ---------------------------------------------------------------------------
template <typename T>
static hipError_t message_impl(const Shape& sh, const Params& pr, const Ws& ws, const void* hidden_v,
                               const void* text_q_v, const void* vis_k_v, const void* probe_v,
                               const float* nonvis_lse, float* trace_omega, float* trace_ebar,
                               hipStream_t st) {
  const T* hidden = static_cast<const T*>(hidden_v);
  timer_mark(kStProbe, true, st);
  hipLaunchKernelGGL(rownorm_kernel<T>, dim3((sh.N + 3) / 4, sh.B), dim3(256), 0, st, sh, ws, hidden);
  RowOperand<T> A{hidden, sh.d, static_cast<long long>(sh.N) * sh.d, nullptr, 0, sh.N};
  RowOperand<T> Bp{static_cast<const T*>(probe_v), sh.d, 0, nullptr, 0, sh.hr};
  ProbeEpi pe{ws, sh.d, pr.rms_eps, sh.hr};
  hipError_t err = launch_gemm_nt<T, 64, 64>(A, Bp, sh.d, sh.B, pe, st);
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(sigma_ell_kernel, dim3(sh.hq, sh.B), dim3(256), 0, st, sh, pr, ws);
  timer_mark(kStProbe, false, st);
  if (sh.T == 0) {
    timer_mark(kStHeads, true, st);
    hipLaunchKernelGGL(no_grounded_kernel, dim3((sh.N + 255) / 256, sh.B), dim3(256), 0, st, sh, ws,
                       trace_omega, trace_ebar);
    timer_mark(kStHeads, false, st);
    return hipGetLastError();
  }
  const dim3 lg((sh.hg * sh.T + 15) / 16, sh.hkv, sh.B);
  const T* q = static_cast<const T*>(text_q_v);
  const T* k = static_cast<const T*>(vis_k_v);
  timer_mark(kStLogits, true, st);
  switch (sh.dh) {
    case 32: hipLaunchKernelGGL((logits_kernel<T, 32>), lg, dim3(256), 0, st, sh, ws, q, k, nonvis_lse); break;
    case 64: hipLaunchKernelGGL((logits_kernel<T, 64>), lg, dim3(256), 0, st, sh, ws, q, k, nonvis_lse); break;
    case 96: hipLaunchKernelGGL((logits_kernel<T, 96>), lg, dim3(256), 0, st, sh, ws, q, k, nonvis_lse); break;
    case 128: hipLaunchKernelGGL((logits_kernel<T, 128>), lg, dim3(256), 0, st, sh, ws, q, k, nonvis_lse); break;
    case 160: hipLaunchKernelGGL((logits_kernel<T, 160>), lg, dim3(256), 0, st, sh, ws, q, k, nonvis_lse); break;
    case 192: hipLaunchKernelGGL((logits_kernel<T, 192>), lg, dim3(256), 0, st, sh, ws, q, k, nonvis_lse); break;
    case 224: hipLaunchKernelGGL((logits_kernel<T, 224>), lg, dim3(256), 0, st, sh, ws, q, k, nonvis_lse); break;
    case 256: hipLaunchKernelGGL((logits_kernel<T, 256>), lg, dim3(256), 0, st, sh, ws, q, k, nonvis_lse); break;
    default: return hipErrorInvalidValue;
  }
  timer_mark(kStLogits, false, st);
  timer_mark(kStHeads, true, st);
  hipLaunchKernelGGL(headgram_kernel, dim3(sh.n_head_blk, sh.B), dim3(256), 0, st, sh, pr, ws);
  hipLaunchKernelGGL(cluster_kernel, dim3(sh.B), dim3(256), 0, st, sh, pr, ws, trace_omega, trace_ebar);
  timer_mark(kStHeads, false, st);
  return hipGetLastError();
}

hipError_t launch_message(const Shape& sh, const Params& pr, const Ws& ws, const void* hidden,
                          const void* text_q, const void* vis_k, const void* probe,
                          const float* nonvis_lse, float* trace_omega, float* trace_ebar,
                          hipStream_t st) {
  if (sh.dtype == 0)
    return message_impl<float>(sh, pr, ws, hidden, text_q, vis_k, probe, nonvis_lse, trace_omega,
                               trace_ebar, st);
  return message_impl<bf16_t>(sh, pr, ws, hidden, text_q, vis_k, probe, nonvis_lse, trace_omega,
                              trace_ebar, st);
}

}  // namespace gmc
