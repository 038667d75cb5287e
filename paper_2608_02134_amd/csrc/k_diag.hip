// Diagnostics of a pruning call, run only when asked for:
//   - the deployed batched-solver certificate of the selection rounds
//     (Prop. 1 Eq. deployed-approximation; App. I Eq. cond-final-cert):
//     U_t = sum of the K largest remaining singleton gains, the round's
//     coverage gain F(S_t u B_t) - F(S_t), q_t = gain / U_t and
//     c_B = 1 - prod_t (1 - q_t), from the gains and pool scores the
//     selection kernels exported and the batches they committed;
//   - the decision margins of each round (relative cut gaps of the pool and
//     the batch);
//   - a scan for non-finite client energies, row weights and outputs
//     (App. J numerical checks);
//   - clearing of the sticky device status bits after the host read them.
#include "gmc_device.h"
#include "gmc_internal.h"
#include "gmc_kernels.h"

namespace gmc {

// Sum of one int per thread over the block.  `red` holds >= 16 ints.
__device__ __forceinline__ int block_sum_int(int v, int* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_sum_i(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  int s = 0;
  for (int i = 0; i < nw; ++i) s += red[i];
  return s;
}

// The k-th largest of n non-negative floats (1 <= k <= n): the largest bit
// pattern c such that at least k values have a pattern >= c (non-negative
// floats order like their bits), found bit by bit from the top.
__device__ float block_kth_largest(const float* v, int n, int k, int* red) {
  uint32_t prefix = 0;
  for (int bit = 30; bit >= 0; --bit) {
    const uint32_t cand = prefix | (1u << bit);
    int c = 0;
    for (int i = threadIdx.x; i < n; i += blockDim.x) c += __float_as_uint(v[i]) >= cand;
    if (block_sum_int(c, red) >= k) prefix = cand;
  }
  return __uint_as_float(prefix);
}

// Relative cut gap (v_(count) - v_(count+1)) / v_(1) of n values; infinite
// when the cut keeps every value or falls between two exact zeros.
__device__ float block_cut_margin(const float* v, int n, int count, int* red) {
  if (count <= 0 || count >= n) return INFINITY;
  const float a = block_kth_largest(v, n, count, red);
  const float b = block_kth_largest(v, n, count + 1, red);
  if (a == 0.f && b == 0.f) return INFINITY;
  const float top = block_kth_largest(v, n, 1, red);
  return top > 0.f ? (a - b) / top : INFINITY;
}

// Coverage gain of every round: one thread per client row walks the rounds'
// batches in order, b_m <- max(b_m, max_{j in B_t} Cbar_mj) with the same
// fp32 products as the selection, and each block stores its sum of
// (new b_m - old b_m) per round.
__global__ void __launch_bounds__(256) cert_cov_kernel(Shape sh, Ws ws, SelOut so) {
  __shared__ float red[16];
  const int p = blockIdx.y, m = blockIdx.x * 256 + threadIdx.x;
  const bool ok = m < sh.m;
  const int mc = ok ? m : 0;
  const float a = ok ? ws.alpha[p * ws.s_m + mc] : 0.f;
  const float* E = ws.E + p * ws.s_E + mc;
  // the rounds start from the image seeds' coverage (none for one image)
  float b = 0.f;
  const int* order = ws.order + p * ws.s_ord;
  for (int g = 0; g < sh.nseed; ++g) b = fmaxf(b, a * E[static_cast<long long>(order[g]) * sh.ldM]);
  int selected = sh.nseed;
  for (int r = 0; r < sh.rounds; ++r) {
    const int bsize = min(sh.b, sh.K - selected);
    const int32_t* bat = so.batch + (static_cast<long long>(p) * sh.rounds + r) * sh.b;
    float c = b;
    for (int k = 0; k < bsize; ++k) c = fmaxf(c, a * E[static_cast<long long>(bat[k]) * sh.ldM]);
    const float d = block_sum(ok ? c - b : 0.f, red);
    if (threadIdx.x == 0) ws.cpart[p * ws.s_cpart + static_cast<long long>(r) * gridDim.x + blockIdx.x] = d;
    b = c;
    selected += bsize;
  }
}

// One block per (round, problem): U_t, the coverage gain, q_t and the two cut
// margins.  Tokens selected before the round carry gain 0, below every
// remaining token, so order statistics over all N equal those over the
// remaining tokens up to their count.
__global__ void __launch_bounds__(256) cert_round_kernel(Shape sh, Ws ws, SelOut so, int ncov_blk) {
  __shared__ float red[16];
  __shared__ int redi[16];
  const int r = blockIdx.x, p = blockIdx.y;
  const int selected = sh.nseed + r * sh.b;
  const int remaining = sh.N - selected;
  const int psize = min(sh.pool_cap, remaining);
  const int bsize = min(sh.b, sh.K - selected);
  const float* u = so.gains + (static_cast<long long>(p) * sh.rounds + r) * sh.N;
  const float* sc = so.scores + (static_cast<long long>(p) * sh.rounds + r) * sh.pool_cap;
  // U_t: the K largest gains (all of them when fewer remain)
  float utop;
  if (remaining <= sh.K) {
    float s = 0.f;
    for (int i = threadIdx.x; i < sh.N; i += blockDim.x) s += u[i];
    utop = block_sum(s, red);
  } else {
    const float thr = block_kth_largest(u, sh.N, sh.K, redi);
    float s = 0.f;
    int c = 0;
    for (int i = threadIdx.x; i < sh.N; i += blockDim.x) {
      const bool gt = u[i] > thr;
      s += gt ? u[i] : 0.f;
      c += gt;
    }
    s = block_sum(s, red);
    c = block_sum_int(c, redi);
    utop = s + static_cast<float>(sh.K - c) * thr;
  }
  const float pool_margin = block_cut_margin(u, sh.N, psize < remaining ? psize : sh.N, redi);
  const float batch_margin = block_cut_margin(sc, psize, bsize, redi);
  float gain = 0.f;
  if (threadIdx.x == 0) {
    const float* cp = ws.cpart + p * ws.s_cpart + static_cast<long long>(r) * ncov_blk;
    for (int k = 0; k < ncov_blk; ++k) gain += cp[k];
    float* ce = ws.cert + p * ws.s_cert + static_cast<long long>(r) * kCertFields;
    ce[0] = utop;
    ce[1] = gain;
    ce[2] = utop > 0.f ? gain / utop : 0.f;
    ce[3] = pool_margin;
    ce[4] = batch_margin;
  }
}

// c_B = 1 - prod_t (1 - q_t), one thread per problem, after the rounds.
__global__ void cert_final_kernel(Shape sh, Ws ws) {
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= sh.B) return;
  float* ce = ws.cert + p * ws.s_cert;
  float prod = 1.f;
  for (int r = 0; r < sh.rounds; ++r) prod *= 1.f - ce[r * kCertFields + 2];
  ce[ws.cert_rounds * kCertFields] = 1.f - prod;
}

hipError_t launch_certificate(const Shape& sh, const Ws& ws, const SelOut& so, hipStream_t st) {
  const int ncov = (sh.m + 255) / 256;
  hipLaunchKernelGGL(cert_cov_kernel, dim3(ncov, sh.B), dim3(256), 0, st, sh, ws, so);
  hipLaunchKernelGGL(cert_round_kernel, dim3(sh.rounds, sh.B), dim3(256), 0, st, sh, ws, so, ncov);
  hipLaunchKernelGGL(cert_final_kernel, dim3((sh.B + 63) / 64), dim3(64), 0, st, sh, ws);
  return hipGetLastError();
}

// Non-finite scan of the weighted client energies alpha_m E[i][m], the row
// weights and the transported outputs; any hit raises the status bit.
template <typename T>
__global__ void __launch_bounds__(256) finite_scan_kernel(Shape sh, Ws ws, const T* out_hidden) {
  const int p = blockIdx.y;
  const long long ne = static_cast<long long>(sh.N) * sh.m;
  const long long no = static_cast<long long>(sh.K) * sh.d;
  const float* E = ws.E + p * ws.s_E;
  const float* alpha = ws.alpha + p * ws.s_m;
  const T* out = out_hidden + p * no;
  bool bad = false;
  const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
  for (long long x = blockIdx.x * static_cast<long long>(blockDim.x) + threadIdx.x; x < ne; x += stride) {
    const int i = static_cast<int>(x / sh.m), m = static_cast<int>(x % sh.m);
    bad |= !isfinite(alpha[m] * E[static_cast<long long>(i) * sh.ldM + m]);
  }
  for (long long x = blockIdx.x * static_cast<long long>(blockDim.x) + threadIdx.x; x < no; x += stride)
    bad |= !isfinite(to_f32(out[x]));
  for (int m = blockIdx.x * blockDim.x + threadIdx.x; m < sh.m; m += static_cast<int>(stride))
    bad |= !isfinite(alpha[m]);
  if (__ballot(bad) != 0ull && (threadIdx.x & 63) == 0) raise_status(ws.cnt + p * ws.s_cnt, kStatusNonfinite);
}

hipError_t launch_finite_scan(const Shape& sh, const Ws& ws, const void* out_hidden, hipStream_t st) {
  const dim3 grid(256, sh.B);
  if (sh.dtype == 0)
    hipLaunchKernelGGL(finite_scan_kernel<float>, grid, dim3(256), 0, st, sh, ws,
                       static_cast<const float*>(out_hidden));
  else
    hipLaunchKernelGGL(finite_scan_kernel<bf16_t>, grid, dim3(256), 0, st, sh, ws,
                       static_cast<const bf16_t*>(out_hidden));
  return hipGetLastError();
}

__global__ void clear_status_kernel(Ws ws, int nprob) {
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p < nprob) __hip_atomic_store(&ws.cnt[p * ws.s_cnt + kCntStatus], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

hipError_t launch_clear_status(const Ws& ws, int nprob, hipStream_t st) {
  hipLaunchKernelGGL(clear_status_kernel, dim3((nprob + 63) / 64), dim3(64), 0, st, ws, nprob);
  return hipGetLastError();
}

}  // namespace gmc
