// Appearance and spatial client banks (Sec. 3.2; App. H Eq. cond-aux-clients,
// Eq. cond-coverage, Eq. cond-effective-bank-mass).
//
// Exact bank (N <= threshold): E_V[m][i] = exp((cos_mi - 1) / tau_v) from an
// MFMA Gram of the raw states, normalised after the contraction
// (cos = h_m.h_i / (|h_m| |h_i|)) so the MFMA operands are the exact inputs.
// The row maximum of x_m.x_i is the self term 1, so no max pass is needed.
// Bounded bank: states projected by the fixed +-1 map, normalised, and
// M_V <= 4096 uniformly spaced clients; the same Gibbs epilogue on the fp32
// projected Gram.  Spatial bank: exp(-(d^2 - min d^2)/tau_s) around the L x L
// landmarks.  Each row keeps its unnormalised energies; the row weight
// alpha_m = (beta_b / M_b) / Z_m folds normalisation and bank mass.
#include "gmc_device.h"
#include "gmc_gemm.h"
#include "gmc_internal.h"
#include "gmc_kernels.h"

namespace gmc {

struct AppearanceEpi {
  Ws ws;
  int ldM;
  int row_off;   // first appearance row of the client matrix
  int exact;     // 1: normalise by row norms; 0: operands already unit
  float inv_tau, norm_eps;
  int ncblk;
  int mv;
  static constexpr bool kRowStats = true;
  // cos = h_m . h_i / (|h_m| |h_i|) on the exact bank (rows are client tokens)
  __device__ float row_scale(int p, int r) const {
    return exact ? 1.f / fmaxf(sqrtf(ws.n2[p * ws.s_n + r]), norm_eps) : 1.f;
  }
  __device__ float col_scale(int p, int c) const {
    return exact ? 1.f / fmaxf(sqrtf(ws.n2[p * ws.s_n + c]), norm_eps) : 1.f;
  }
  __device__ float value(int p, int r, int c, float cs) const {
    const float v = expf((cs - 1.f) * inv_tau);
    ws.E[p * ws.s_E + static_cast<long long>(c) * ldM + row_off + r] = v;
    return v;
  }
  __device__ void row_stats(int p, int r, int cblk, float s, float m) const {
    ws.apart_sum[p * ws.s_apart + static_cast<long long>(cblk) * mv + r] = s;
    ws.apart_max[p * ws.s_apart + static_cast<long long>(cblk) * mv + r] = m;
  }
};

// Bounded bank: raw projection y = R h (fp32 out).
struct ProjEpi {
  Ws ws;
  int rank;
  static constexpr bool kRowStats = false;
  __device__ float row_scale(int, int) const { return 1.f; }
  __device__ float col_scale(int, int) const { return 1.f; }
  __device__ float value(int p, int r, int c, float v) const {
    ws.y[p * ws.s_y + static_cast<long long>(r) * rank + c] = v;
    return v;
  }
  __device__ void row_stats(int, int, int, float, float) const {}
};

// Normalise projected rows: one wave per token.
__global__ void __launch_bounds__(256) normalize_rows_kernel(Shape sh, Params pr, Ws ws) {
  const int p = blockIdx.y, i = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (i >= sh.N) return;
  float* y = ws.y + p * ws.s_y + static_cast<long long>(i) * sh.app_rank;
  float s = 0.f;
  for (int c = lane; c < sh.app_rank; c += 64) s += y[c] * y[c];
  s = wave_sum(s);
  const float inv = 1.f / fmaxf(sqrtf(s), pr.norm_eps);
  for (int c = lane; c < sh.app_rank; c += 64) y[c] *= inv;
}

// Client tokens m_k = floor(k N / M_V) of the bounded bank.
__global__ void clients_kernel(Shape sh, Ws ws) {
  const int p = blockIdx.y;
  for (int k = blockIdx.x * blockDim.x + threadIdx.x; k < sh.mv; k += gridDim.x * blockDim.x)
    ws.clients[p * ws.s_cl + k] =
        static_cast<int>((static_cast<long long>(k) * sh.N) / sh.mv);
}

// Appearance row weights alpha = (beta_app / M_V) / Z_m and peaks.
__global__ void __launch_bounds__(256) appearance_alpha_kernel(Shape sh, Params pr, Ws ws) {
  const int p = blockIdx.y;
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= sh.mv) return;
  const float* ps = ws.apart_sum + p * ws.s_apart;
  const float* pm = ws.apart_max + p * ws.s_apart;
  float s = 0.f, m = 0.f;
#pragma unroll 8
  for (int b = 0; b < sh.n_app_cblk; ++b) {
    s += ps[static_cast<long long>(b) * sh.mv + r];
    m = fmaxf(m, pm[static_cast<long long>(b) * sh.mv + r]);
  }
  const float a = pr.beta_app / static_cast<float>(sh.mv) / s;
  ws.alpha[p * ws.s_m + sh.mg + r] = a;
  ws.peak[p * ws.s_m + sh.mg + r] = a * m;
}

// Grid origin/extent of (h, w) and the per-token spatial coordinates,
// cell centres in [0,1]^2 (temporal id excluded).
__global__ void __launch_bounds__(256) spatial_coords_kernel(Shape sh, Ws ws, const int32_t* pos3d) {
  __shared__ float red[16];
  const int p = blockIdx.x;
  const int32_t* pos = pos3d + static_cast<long long>(p) * sh.N * 3;
  float hmin = INFINITY, hmax = -INFINITY, wmin = INFINITY, wmax = -INFINITY;
  for (int i = threadIdx.x; i < sh.N; i += blockDim.x) {
    const float hh = static_cast<float>(pos[i * 3 + 1]), ww = static_cast<float>(pos[i * 3 + 2]);
    hmin = fminf(hmin, hh); hmax = fmaxf(hmax, hh);
    wmin = fminf(wmin, ww); wmax = fmaxf(wmax, ww);
  }
  hmin = block_min(hmin, red);
  hmax = block_max(hmax, red);
  wmin = block_min(wmin, red);
  wmax = block_max(wmax, red);
  const float gh = hmax - hmin + 1.f, gw = wmax - wmin + 1.f;
  float* pc = ws.pc + p * ws.s_pc;
  for (int i = threadIdx.x; i < sh.N; i += blockDim.x) {
    pc[2 * i] = (static_cast<float>(pos[i * 3 + 1]) - hmin + 0.5f) / gh;
    pc[2 * i + 1] = (static_cast<float>(pos[i * 3 + 2]) - wmin + 0.5f) / gw;
  }
}

// Spatial bank, landmark side: one block per landmark l_ab = ((a+.5)/L,
// (b+.5)/L): the minimum squared distance to any token, the row sum of
// exp(-(d^2 - min d^2)/tau_s), the weight (beta_spa / L^2) / Z and the peak
// (the row maximum is exactly 1).
__global__ void __launch_bounds__(256) spatial_stats_kernel(Shape sh, Params pr, Ws ws) {
  __shared__ float red[16];
  const int row = blockIdx.x, p = blockIdx.y;
  const int L = sh.landmarks;
  const float ly = (static_cast<float>(row / L) + 0.5f) / L;
  const float lx = (static_cast<float>(row % L) + 0.5f) / L;
  const float* pc = ws.pc + p * ws.s_pc;
  float dmin = INFINITY;
  for (int i = threadIdx.x; i < sh.N; i += blockDim.x) {
    const float dy = pc[2 * i] - ly, dx = pc[2 * i + 1] - lx;
    dmin = fminf(dmin, dy * dy + dx * dx);
  }
  dmin = block_min(dmin, red);
  const float inv_tau = 1.f / pr.tau_s;
  float s = 0.f;
  for (int i = threadIdx.x; i < sh.N; i += blockDim.x) {
    const float dy = pc[2 * i] - ly, dx = pc[2 * i + 1] - lx;
    s += expf(-(dy * dy + dx * dx - dmin) * inv_tau);
  }
  s = block_sum(s, red);
  if (threadIdx.x == 0) {
    const int m = sh.mg + sh.mv + row;
    const float a = pr.beta_spa / static_cast<float>(sh.ms) / s;
    ws.alpha[p * ws.s_m + m] = a;
    ws.peak[p * ws.s_m + m] = a;
    ws.lstat[p * ws.s_lstat + row] = dmin;
  }
}

// Spatial bank, token side: one wave per token writes its L^2 landmark
// energies, contiguous in the token-major client matrix.
__global__ void __launch_bounds__(256) spatial_write_kernel(Shape sh, Params pr, Ws ws) {
  const int p = blockIdx.y, i = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (i >= sh.N) return;
  const int L = sh.landmarks;
  const float* pc = ws.pc + p * ws.s_pc;
  const float py = pc[2 * i], px = pc[2 * i + 1];
  const float inv_tau = 1.f / pr.tau_s;
  const float* dmin = ws.lstat + p * ws.s_lstat;
  float* E = ws.E + p * ws.s_E + static_cast<long long>(i) * sh.ldM + sh.mg + sh.mv;
  for (int row = lane; row < sh.ms; row += 64) {
    const float ly = (static_cast<float>(row / L) + 0.5f) / L;
    const float lx = (static_cast<float>(row % L) + 0.5f) / L;
    const float dy = py - ly, dx = px - lx;
    E[row] = expf(-(dy * dy + dx * dx - dmin[row]) * inv_tau);
  }
}

template <typename T>
static hipError_t banks_impl(const Shape& sh, const Params& pr, const Ws& ws, const void* hidden_v,
                             const void* proj_v, const int32_t* pos3d, hipStream_t st) {
  const T* hidden = static_cast<const T*>(hidden_v);
  hipError_t err;
  timer_mark(kStAppearance, true, st);
  if (!sh.bounded) {
    RowOperand<T> A{hidden, sh.d, static_cast<long long>(sh.N) * sh.d, nullptr, 0, sh.N};
    AppearanceEpi epi{ws, sh.ldM, sh.mg, 1, 1.f / pr.tau_v, pr.norm_eps, sh.n_app_cblk, sh.mv};
    err = launch_gemm_nt<T, 64, 64>(A, A, sh.d, sh.B, epi, st);
    if (err != hipSuccess) return err;
  } else {
    RowOperand<T> A{hidden, sh.d, static_cast<long long>(sh.N) * sh.d, nullptr, 0, sh.N};
    RowOperand<T> R{static_cast<const T*>(proj_v), sh.d, 0, nullptr, 0, sh.app_rank};
    ProjEpi pe{ws, sh.app_rank};
    err = launch_gemm_nt<T, 64, 64>(A, R, sh.d, sh.B, pe, st);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(normalize_rows_kernel, dim3((sh.N + 3) / 4, sh.B), dim3(256), 0, st, sh, pr, ws);
    hipLaunchKernelGGL(clients_kernel, dim3((sh.mv + 255) / 256, sh.B), dim3(256), 0, st, sh, ws);
    RowOperand<float> Yc{ws.y, sh.app_rank, ws.s_y, ws.clients, ws.s_cl, sh.mv};
    RowOperand<float> Y{ws.y, sh.app_rank, ws.s_y, nullptr, 0, sh.N};
    AppearanceEpi epi{ws, sh.ldM, sh.mg, 0, 1.f / pr.tau_v, pr.norm_eps, sh.n_app_cblk, sh.mv};
    err = launch_gemm_nt<float, 64, 64>(Yc, Y, sh.app_rank, sh.B, epi, st);
    if (err != hipSuccess) return err;
  }
  timer_mark(kStAppearance, false, st);
  timer_mark(kStSpatial, true, st);
  hipLaunchKernelGGL(appearance_alpha_kernel, dim3((sh.mv + 255) / 256, sh.B), dim3(256), 0, st, sh, pr, ws);
  hipLaunchKernelGGL(spatial_coords_kernel, dim3(sh.B), dim3(256), 0, st, sh, ws, pos3d);
  hipLaunchKernelGGL(spatial_stats_kernel, dim3(sh.ms, sh.B), dim3(256), 0, st, sh, pr, ws);
  hipLaunchKernelGGL(spatial_write_kernel, dim3((sh.N + 3) / 4, sh.B), dim3(256), 0, st, sh, pr, ws);
  timer_mark(kStSpatial, false, st);
  return hipGetLastError();
}

hipError_t launch_banks(const Shape& sh, const Params& pr, const Ws& ws, const void* hidden,
                        const void* app_proj, const int32_t* pos3d, hipStream_t st) {
  if (sh.dtype == 0) return banks_impl<float>(sh, pr, ws, hidden, app_proj, pos3d, st);
  return banks_impl<bf16_t>(sh, pr, ws, hidden, app_proj, pos3d, st);
}

}  // namespace gmc
