// Batched responsibility selection (Sec. 3.3 Eq. coverage, Eq.
// responsibility; App. H Eq. cond-responsibility and the totality rule).
//
// Client row m has weight alpha_m and energies E_m, so Cbar_mi = alpha_m E_mi
// is formed on the fly; coverage maxima b_m live in a ping-pong pair.  One
// round is four kernels:
//   gains  - refresh b_m with the previous batch, then partial column sums of
//            R_mi = [Cbar_mi - b_m]_+ over row chunks (float4 streaming)
//   pool   - one block per problem: fixed-order sum of the partials, then a
//            deterministic radix top-k of (gain desc, index asc) over the
//            unselected tokens
//   resp   - responsibility softmax of R over the pool per client row,
//            partial column sums of rho R over row chunks
//   batch  - one block per problem: top-b of the pool scores, mark them
// Every reduction has a fixed order, so results are bitwise repeatable.
// Zero-gain tokens key just above excluded ones, so once gains vanish the
// lowest source indices fill the budget.
#include "gmc_device.h"
#include "gmc_internal.h"
#include "gmc_kernels.h"

namespace gmc {

constexpr int kSubRows = 256;

__global__ void __launch_bounds__(256) gains_kernel(Shape sh, Ws ws, int round, int prev_b) {
  __shared__ float cov_s[kSubRows];
  __shared__ float4 wsum[4][64];
  const int p = blockIdx.y;
  const int strip = blockIdx.x % sh.nstrips, chunk = blockIdx.x / sh.nstrips;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r0 = chunk * sh.rc, r1 = min(sh.m, r0 + sh.rc);
  const float* cov_in = ws.cov + p * ws.s_cov + (round & 1) * sh.m;
  float* cov_out = ws.cov + p * ws.s_cov + ((round + 1) & 1) * sh.m;
  const int* prev = ws.batch + p * ws.s_bat;
  const float* E = ws.E + p * ws.s_E;
  const float* alpha = ws.alpha + p * ws.s_m;
  const int c0 = strip * kStripCols + lane * 4;
  const bool col_ok = c0 < sh.N;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s0 = r0; s0 < r1; s0 += kSubRows) {
    const int n = min(kSubRows, r1 - s0);
    __syncthreads();
    if (tid < n) {
      const int m = s0 + tid;
      const float a = alpha[m];
      float c = (round == 0) ? 0.f : cov_in[m];
      const float* Em = E + static_cast<long long>(m) * sh.ldE;
      for (int j = 0; j < prev_b; ++j) c = fmaxf(c, a * Em[prev[j]]);
      cov_s[tid] = c;
      if (strip == 0) cov_out[m] = c;
    }
    __syncthreads();
    if (col_ok) {
      for (int rr = wave; rr < n; rr += 4) {
        const int m = s0 + rr;
        const float a = alpha[m], c = cov_s[rr];
        const float4 v = *reinterpret_cast<const float4*>(E + static_cast<long long>(m) * sh.ldE + c0);
        acc.x += fmaxf(a * v.x - c, 0.f);
        acc.y += fmaxf(a * v.y - c, 0.f);
        acc.z += fmaxf(a * v.z - c, 0.f);
        acc.w += fmaxf(a * v.w - c, 0.f);
      }
    }
  }
  wsum[wave][lane] = acc;
  __syncthreads();
  if (wave == 0 && col_ok) {
    float4 s = wsum[0][lane];
    for (int w = 1; w < 4; ++w) {
      const float4 t = wsum[w][lane];
      s.x += t.x; s.y += t.y; s.z += t.z; s.w += t.w;
    }
    *reinterpret_cast<float4*>(ws.part + p * ws.s_part + static_cast<long long>(chunk) * sh.ldE + c0) = s;
  }
}

// Deterministic block top-k over n keys held in LDS: the `count` largest
// keys, equal keys resolved to the lower index.  Indices are written in
// ascending order to out[0..count).  count must not exceed the number of
// non-zero keys.  Uses radix selection of the threshold key (4 passes of
// 8-bit digits) and ordered compaction in rounds of blockDim.x indices.
__device__ void block_topk(const uint32_t* keys, int n, int count, int* out, int* hist, int* scan,
                           int* bcast) {
  const int tid = threadIdx.x, nt = blockDim.x;
  uint32_t prefix = 0, mask = 0;
  int remaining = count;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int b = tid; b < 256; b += nt) hist[b] = 0;
    __syncthreads();
    for (int i = tid; i < n; i += nt) {
      const uint32_t k = keys[i];
      if ((k & mask) == prefix) atomicAdd(&hist[(k >> shift) & 255u], 1);
    }
    __syncthreads();
    if (tid == 0) {
      int cum = 0, d = 255;
      for (; d > 0; --d) {
        if (cum + hist[d] >= remaining) break;
        cum += hist[d];
      }
      bcast[0] = d;
      bcast[1] = remaining - cum;
    }
    __syncthreads();
    prefix |= static_cast<uint32_t>(bcast[0]) << shift;
    mask |= 0xFFu << shift;
    remaining = bcast[1];
    __syncthreads();
  }
  const uint32_t kth = prefix;
  int eq_seen = 0, written = 0;
  for (int b0 = 0; b0 < n; b0 += nt) {
    const int i = b0 + tid;
    const uint32_t k = (i < n) ? keys[i] : 0u;
    const int is_eq = (i < n && k == kth) ? 1 : 0;
    int eq_tot;
    const int eq_before = eq_seen + block_exclusive_scan(is_eq, scan, &eq_tot);
    const int take = (i < n) && (k > kth || (is_eq && eq_before < remaining));
    int tot;
    const int pos = written + block_exclusive_scan(take, scan, &tot);
    if (take) out[pos] = i;
    eq_seen += eq_tot;
    written += tot;
  }
  __syncthreads();
}

// Keys live in LDS when N fits (kLdsKeys), else in the workspace (L2).
constexpr int kLdsKeys = 12288;

template <bool kGlobalKeys>
__global__ void __launch_bounds__(1024) pool_kernel(Shape sh, Ws ws, int round, int psize,
                                                    int32_t* trace_pool) {
  extern __shared__ uint32_t keys_lds[];
  __shared__ int hist[256], scan[16], bcast[2];
  const int p = blockIdx.x, tid = threadIdx.x;
  uint32_t* keys = kGlobalKeys ? ws.keys + p * ws.s_keys : keys_lds;
  const float* part = ws.part + p * ws.s_part;
  const int* sel = ws.sel + p * ws.s_sel;
  for (int i = tid; i < sh.N; i += blockDim.x) {
    float u = 0.f;
    for (int c = 0; c < sh.nc; ++c) u += part[static_cast<long long>(c) * sh.ldE + i];
    keys[i] = (sel[i] >= 0) ? 0u : score_key(u);
  }
  __syncthreads();
  int* pool = ws.pool + p * ws.s_pool;
  block_topk(keys, sh.N, psize, pool, hist, scan, bcast);
  if (trace_pool) {
    int32_t* tp = trace_pool + (static_cast<long long>(p) * sh.rounds + round) * sh.pool_cap;
    for (int j = tid; j < sh.pool_cap; j += blockDim.x) tp[j] = (j < psize) ? pool[j] : -1;
  }
}

template <int Q>
__global__ void __launch_bounds__(256) resp_kernel(Shape sh, Params pr, Ws ws, int round, int psize) {
  __shared__ int pool_s[64 * Q];
  __shared__ float acc_s[4][64 * Q];
  const int p = blockIdx.y, chunk = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int* pool = ws.pool + p * ws.s_pool;
  for (int j = tid; j < 64 * Q; j += 256) pool_s[j] = (j < psize) ? pool[j] : 0;
  __syncthreads();
  const float* cov = ws.cov + p * ws.s_cov + ((round + 1) & 1) * sh.m;
  const float* E = ws.E + p * ws.s_E;
  const float* alpha = ws.alpha + p * ws.s_m;
  float racc[Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) racc[q] = 0.f;
  const int r0 = chunk * sh.rc2, r1 = min(sh.m, r0 + sh.rc2);
  for (int m = r0 + wave; m < r1; m += 4) {
    const float a = alpha[m], c = cov[m];
    const float* Em = E + static_cast<long long>(m) * sh.ldE;
    float R[Q];
    float mu = 0.f;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int jj = lane + 64 * q;
      R[q] = (jj < psize) ? fmaxf(a * Em[pool_s[jj]] - c, 0.f) : 0.f;
      mu = fmaxf(mu, R[q]);
    }
    mu = wave_max(mu);
    if (mu > 0.f) {
      const float inv = 1.f / (pr.tau_r * mu + pr.resp_eps);
      const float zmax = mu * inv;
      float ex[Q];
      float den = 0.f;
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        const int jj = lane + 64 * q;
        ex[q] = (jj < psize) ? expf(R[q] * inv - zmax) : 0.f;
        den += ex[q];
      }
      den = wave_sum(den);
      const float rden = 1.f / den;
#pragma unroll
      for (int q = 0; q < Q; ++q) racc[q] += ex[q] * rden * R[q];
    }
  }
#pragma unroll
  for (int q = 0; q < Q; ++q) acc_s[wave][lane + 64 * q] = racc[q];
  __syncthreads();
  float* sp = ws.spart + p * ws.s_spart + static_cast<long long>(chunk) * sh.pool_cap;
  for (int j = tid; j < psize; j += 256) sp[j] = ((acc_s[0][j] + acc_s[1][j]) + acc_s[2][j]) + acc_s[3][j];
}

__global__ void __launch_bounds__(1024) batch_kernel(Shape sh, Ws ws, int round, int psize, int bsize,
                                                     int sel_base, int32_t* trace_batch) {
  extern __shared__ uint32_t keys[];
  __shared__ int hist[256], scan[16], bcast[2];
  __shared__ int chosen[1024];
  const int p = blockIdx.x, tid = threadIdx.x;
  const float* sp = ws.spart + p * ws.s_spart;
  for (int j = tid; j < psize; j += blockDim.x) {
    float s = 0.f;
    for (int c = 0; c < sh.nc2; ++c) s += sp[static_cast<long long>(c) * sh.pool_cap + j];
    keys[j] = score_key(s);
  }
  __syncthreads();
  block_topk(keys, psize, bsize, chosen, hist, scan, bcast);
  const int* pool = ws.pool + p * ws.s_pool;
  int* sel = ws.sel + p * ws.s_sel;
  int* order = ws.order + p * ws.s_ord;
  int* batch = ws.batch + p * ws.s_bat;
  for (int k = tid; k < bsize; k += blockDim.x) {
    const int i = pool[chosen[k]];
    sel[i] = round;
    order[sel_base + k] = i;
    batch[k] = i;
  }
  if (trace_batch) {
    int32_t* tb = trace_batch + (static_cast<long long>(p) * sh.rounds + round) * sh.b;
    for (int k = tid; k < sh.b; k += blockDim.x) tb[k] = (k < bsize) ? pool[chosen[k]] : -1;
  }
}

// Initial state: nothing selected.
__global__ void select_init_kernel(Shape sh, Ws ws) {
  const int p = blockIdx.y;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < sh.N; i += gridDim.x * blockDim.x)
    ws.sel[p * ws.s_sel + i] = -1;
}

// Final coverage b_m(S) and per-block partial sums of F(S) and F(V).
__global__ void __launch_bounds__(256) cov_final_kernel(Shape sh, Ws ws, int last_b) {
  __shared__ float red[16];
  const int p = blockIdx.y, m = blockIdx.x * 256 + threadIdx.x;
  const float* cov_in = ws.cov + p * ws.s_cov + (sh.rounds & 1) * sh.m;
  const int* prev = ws.batch + p * ws.s_bat;
  float c = 0.f, pk = 0.f;
  if (m < sh.m) {
    const float a = ws.alpha[p * ws.s_m + m];
    c = cov_in[m];
    const float* Em = ws.E + p * ws.s_E + static_cast<long long>(m) * sh.ldE;
    for (int j = 0; j < last_b; ++j) c = fmaxf(c, a * Em[prev[j]]);
    pk = ws.peak[p * ws.s_m + m];
  }
  const float fs = block_sum(c, red);
  const float fv = block_sum(pk, red);
  if (threadIdx.x == 0) {
    ws.spart[p * ws.s_spart + 2 * blockIdx.x] = fs;
    ws.spart[p * ws.s_spart + 2 * blockIdx.x + 1] = fv;
  }
}

__global__ void objective_stats_kernel(Shape sh, Ws ws, int nblk) {
  const int p = blockIdx.x;
  if (threadIdx.x != 0) return;
  float fs = 0.f, fv = 0.f;
  for (int b = 0; b < nblk; ++b) {
    fs += ws.spart[p * ws.s_spart + 2 * b];
    fv += ws.spart[p * ws.s_spart + 2 * b + 1];
  }
  float* st = ws.stats + p * ws.s_st;
  st[2] = fs;
  st[3] = fv;
  st[4] = static_cast<float>(sh.K);
  st[5] = static_cast<float>(sh.rounds);
  st[6] = static_cast<float>(sh.m);
  st[7] = static_cast<float>(sh.N - sh.K);
}

hipError_t launch_selection(const Shape& sh, const Params& pr, const Ws& ws, int32_t* trace_pool,
                            int32_t* trace_batch, hipStream_t st) {
  hipLaunchKernelGGL(select_init_kernel, dim3((sh.N + 255) / 256, sh.B), dim3(256), 0, st, sh, ws);
  const size_t pool_lds = static_cast<size_t>(sh.N) * sizeof(uint32_t);
  const size_t batch_lds = static_cast<size_t>(sh.pool_cap) * sizeof(uint32_t);
  int selected = 0;
  for (int r = 0; r < sh.rounds; ++r) {
    const int psize = min(sh.pool_cap, sh.N - selected);
    const int bsize = min(sh.b, sh.K - selected);
    timer_mark(kStGains, true, st);
    hipLaunchKernelGGL(gains_kernel, dim3(sh.nstrips * sh.nc, sh.B), dim3(256), 0, st, sh, ws, r,
                       r > 0 ? sh.b : 0);
    timer_mark(kStGains, false, st);
    timer_mark(kStPool, true, st);
    if (sh.N <= kLdsKeys)
      hipLaunchKernelGGL(pool_kernel<false>, dim3(sh.B), dim3(1024), pool_lds, st, sh, ws, r, psize, trace_pool);
    else
      hipLaunchKernelGGL(pool_kernel<true>, dim3(sh.B), dim3(1024), 0, st, sh, ws, r, psize, trace_pool);
    timer_mark(kStPool, false, st);
    timer_mark(kStResp, true, st);
    const int q = (sh.pool_cap + 63) / 64;
    const dim3 rg(sh.nc2, sh.B);
    if (q <= 1) hipLaunchKernelGGL(resp_kernel<1>, rg, dim3(256), 0, st, sh, pr, ws, r, psize);
    else if (q <= 2) hipLaunchKernelGGL(resp_kernel<2>, rg, dim3(256), 0, st, sh, pr, ws, r, psize);
    else if (q <= 4) hipLaunchKernelGGL(resp_kernel<4>, rg, dim3(256), 0, st, sh, pr, ws, r, psize);
    else if (q <= 8) hipLaunchKernelGGL(resp_kernel<8>, rg, dim3(256), 0, st, sh, pr, ws, r, psize);
    else if (q <= 16) hipLaunchKernelGGL(resp_kernel<16>, rg, dim3(256), 0, st, sh, pr, ws, r, psize);
    else if (q <= 32) hipLaunchKernelGGL(resp_kernel<32>, rg, dim3(256), 0, st, sh, pr, ws, r, psize);
    else return hipErrorInvalidValue;
    timer_mark(kStResp, false, st);
    timer_mark(kStBatch, true, st);
    hipLaunchKernelGGL(batch_kernel, dim3(sh.B), dim3(1024), batch_lds, st, sh, ws, r, psize, bsize,
                       selected, trace_batch);
    timer_mark(kStBatch, false, st);
    selected += bsize;
  }
  const int last_b = sh.K - (sh.rounds - 1) * sh.b;
  const int nblk = (sh.m + 255) / 256;
  timer_mark(kStObjective, true, st);
  hipLaunchKernelGGL(cov_final_kernel, dim3(nblk, sh.B), dim3(256), 0, st, sh, ws, last_b);
  hipLaunchKernelGGL(objective_stats_kernel, dim3(sh.B), dim3(64), 0, st, sh, ws, nblk);
  timer_mark(kStObjective, false, st);
  return hipGetLastError();
}

}  // namespace gmc
