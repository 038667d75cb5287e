// Population assignment (Sec. 3.4; App. H Eq. cond-assignment, Eq.
// cond-population-gate).
//
// cos_ij = h_i.h_j / (|h_i| |h_j|) for every token i and support member j.
// With the exact appearance bank every pair's cosine is already stored as
// E_V = exp((cos - 1) / tau_v) in the client matrix (client row j, token i),
// so cos_ij = 1 + tau_v ln E_V is gathered from there; the bounded bank keeps
// only projected cosines, so there an MFMA GEMM against the gathered support
// rows (normalised after the contraction) computes them.  The gap delta_i (best - second best), the sample gate
// s_x = 1 - exp(-(mean_discarded delta / t)^p) and the local ambiguity g_i
// then decide kappa_ij = cos_ij + w s_x g_i exp(-|p_i - p_j|^2 / tau_s);
// pi(i) = argmax_j kappa_ij with ties to the lower source index, and
// selected tokens represent themselves.
#include "gmc_device.h"
#include "gmc_gemm.h"
#include "gmc_internal.h"
#include "gmc_kernels.h"

namespace gmc {

// Support in ascending source order and each selected token's slot.
__global__ void __launch_bounds__(1024) support_kernel(Shape sh, Ws ws) {
  __shared__ int scan[16];
  const int p = blockIdx.x, tid = threadIdx.x;
  const int* sel = ws.sel + p * ws.s_sel;
  int* slot = ws.slot + p * ws.s_slot;
  int* sup = ws.sup + p * ws.s_sup;
  int base = 0;
  for (int b0 = 0; b0 < sh.N; b0 += blockDim.x) {
    const int i = b0 + tid;
    const int f = (i < sh.N && sel[i] >= 0) ? 1 : 0;
    int tot;
    const int pos = base + block_exclusive_scan(f, scan, &tot);
    if (i < sh.N) {
      slot[i] = f ? pos : -1;
      if (f) sup[pos] = i;
    }
    base += tot;
  }
}

struct CosEpi {
  Ws ws;
  int ldK;
  float norm_eps;
  static constexpr bool kRowStats = false;
  __device__ float row_scale(int p, int r) const {
    return 1.f / fmaxf(sqrtf(ws.n2[p * ws.s_n + r]), norm_eps);
  }
  __device__ float col_scale(int p, int c) const {
    return 1.f / fmaxf(sqrtf(ws.n2[p * ws.s_n + ws.sup[p * ws.s_sup + c]]), norm_eps);
  }
  __device__ float value(int p, int r, int c, float v) const {
    ws.cosb[p * ws.s_cos + static_cast<long long>(r) * ldK + c] = v;
    return v;
  }
  __device__ void row_stats(int, int, int, float, float) const {}
};

// Cosine of token i to the support member in slot j: from the stored
// appearance client value (exact bank) or from the GEMM output.
template <bool kFromE>
struct CosSource {
  const float* row;   // E row of token i (kFromE) or cosb row of token i
  int mg;
  const int* sup;
  float tau_v;
  __device__ __forceinline__ float get(int j) const {
    if constexpr (kFromE) return 1.f + tau_v * __logf(row[mg + sup[j]]);
    else return row[j];
  }
};

template <bool kFromE>
__device__ __forceinline__ CosSource<kFromE> cos_source(const Shape& sh, const Params& pr, const Ws& ws, int p, int i) {
  CosSource<kFromE> c;
  c.row = kFromE ? ws.E + p * ws.s_E + static_cast<long long>(i) * sh.ldM
                 : ws.cosb + p * ws.s_cos + static_cast<long long>(i) * sh.ldK;
  c.mg = sh.mg;
  c.sup = ws.sup + p * ws.s_sup;
  c.tau_v = pr.tau_v;
  return c;
}

// delta_i = top1 - top2 of cos_i. over the support (0 when K = 1), and the
// token's grounded energy e_i = sqrt(sum_h omega_h sum_t nu_t e^2) (Eq.
// cond-grounded-energy; the head-pattern kernel left sum_t nu_t e^2 per head);
// one wave per token.

// One butterfly step of a wave-wide (largest, second largest) pair.
template <int O>
__device__ __forceinline__ void top2_step(float& t1, float& t2) {
  const float o1 = xor_lane<O>(t1), o2 = xor_lane<O>(t2);
  const float n1 = fmaxf(t1, o1);
  const float n2 = fmaxf(fminf(t1, o1), fmaxf(t2, o2));
  t1 = n1;
  t2 = n2;
}
// One butterfly step of a wave-wide argmax (ties to the lower index).
template <int O>
__device__ __forceinline__ void argmax_step(float& best, int& bj) {
  const float ob = xor_lane<O>(best);
  const int oj = xor_lane_i<O>(bj);
  if (ob > best || (ob == best && oj < bj)) { best = ob; bj = oj; }
}

template <bool kFromE>
__global__ void __launch_bounds__(256) gap_kernel(Shape sh, Params pr, Ws ws) {
  const int p = blockIdx.y, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = blockIdx.x * 4 + wave;
  if (i < sh.N) {
    // the energy inputs go out with the first cosine loads
    const float w = (sh.T > 0 && lane < sh.hq)
                        ? ws.omega[p * ws.s_om + lane] * ws.e2[p * ws.s_e2 + static_cast<long long>(lane) * sh.N + i]
                        : 0.f;
    const CosSource<kFromE> cs = cos_source<kFromE>(sh, pr, ws, p, i);
    float t1 = -INFINITY, t2 = -INFINITY;
    for (int j0 = 0; j0 < sh.K; j0 += 64 * 8) {
      float v[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = cs.get(min(j0 + q * 64 + lane, sh.K - 1));
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        if (j0 + q * 64 + lane >= sh.K) continue;
        if (v[q] > t1) { t2 = t1; t1 = v[q]; }
        else if (v[q] > t2) t2 = v[q];
      }
    }
    top2_step<32>(t1, t2);
    top2_step<16>(t1, t2);
    top2_step<8>(t1, t2);
    top2_step<4>(t1, t2);
    top2_step<2>(t1, t2);
    top2_step<1>(t1, t2);
    // no second compatible carrier (K = 1, or the token's image has one
    // carrier and the others read -inf): the gap is 0
    const float delta = (sh.K >= 2 && t2 > -INFINITY) ? t1 - t2 : 0.f;
    if (lane == 0) ws.delta[p * ws.s_del + i] = delta;
    if (sh.T > 0) {
      // lane h holds head h (at most kMaxHeads of them)
      const float e = sqrtf(wave_sum(w));
      if (lane == 0) ws.ebar[p * ws.s_eb + i] = e;
    }
  }
}

// The separability gate s_x = 1 - exp(-(mean delta / t)^p) over the discarded
// tokens and 1 / mean e (the population weights' normaliser; 0 selects the
// uniform fallback ebar = 1), formed by every block from all tokens (a fixed
// summation order, so every block holds the same values); block 0 records
// them.
__device__ float separability_gate(const Shape& sh, const Params& pr, const Ws& ws, int p, float* red) {
  const float* delta = ws.delta + p * ws.s_del;
  const float* eb = ws.ebar + p * ws.s_eb;
  const int* sel = ws.sel + p * ws.s_sel;
  float s = 0.f, se = 0.f;
  for (int i0 = 0; i0 < sh.N; i0 += 256 * 8) {
    float dv[8], ev[8];
    int sv[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int i = min(i0 + q * 256 + static_cast<int>(threadIdx.x), sh.N - 1);
      dv[q] = delta[i];
      ev[q] = eb[i];
      sv[q] = sel[i];
    }
#pragma unroll
    for (int q = 0; q < 8; ++q)
      if (i0 + q * 256 + static_cast<int>(threadIdx.x) < sh.N) {
        if (sv[q] < 0) s += dv[q];
        se += ev[q];
      }
  }
  s = block_sum(s, red);
  se = block_sum(se, red);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    const float mean = se / static_cast<float>(sh.N);
    ws.gate[p * ws.s_gate + 2] = mean > 0.f ? 1.f / mean : 0.f;
  }
  const int nd = sh.N - sh.K;
  const float dbar = nd > 0 ? s / static_cast<float>(nd) : 0.f;
  const float sx = 1.f - expf(-powf(dbar / pr.gate_t, pr.gate_p));
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    ws.gate[p * ws.s_gate + 0] = sx;
    ws.gate[p * ws.s_gate + 1] = dbar;
    ws.stats[p * ws.s_st + 0] = sx;
    ws.stats[p * ws.s_st + 1] = dbar;
  }
  return sx;
}

// pi(i) = argmax_j kappa_ij; one wave per token.
template <bool kFromE>
__global__ void __launch_bounds__(256) kappa_kernel(Shape sh, Params pr, Ws ws, int32_t* trace_assign) {
  __shared__ float red[16];
  const int p = blockIdx.y, lane = threadIdx.x & 63;
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int ic = min(i, sh.N - 1);
  const int* sup = ws.sup + p * ws.s_sup;
  const float* pc = ws.pc + p * ws.s_pc;
  const CosSource<kFromE> cs = cos_source<kFromE>(sh, pr, ws, p, ic);
  // the token's own loads and its first support batch (cosines and spatial
  // coordinates) go out before the gate's block reductions
  const bool selected = ws.sel[p * ws.s_sel + ic] >= 0;
  const float delta = ws.delta[p * ws.s_del + ic];
  const float py = pc[2 * ic], px = pc[2 * ic + 1];
  float c0[4], y0[4], x0[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int j = min(q * 64 + lane, sh.K - 1);
    const int sj = sup[j];
    c0[q] = cs.get(j);
    y0[q] = pc[2 * sj];
    x0[q] = pc[2 * sj + 1];
  }
  const float sx = separability_gate(sh, pr, ws, p, red);
  if (i >= sh.N) return;
  int pi_i;
  if (selected) {
    pi_i = i;
  } else {
    const float g = (pr.g_form == 1) ? (delta < pr.amb_margin ? 1.f : 0.f)
                                     : expf(-powf(delta / pr.amb_margin, pr.amb_p));
    const float w = pr.spatial_w * sx * g;
    const float inv_tau = 1.f / pr.tau_s;
    float best = -INFINITY;
    int bj = 0x7fffffff;
    for (int j0 = 0; j0 < sh.K; j0 += 64 * 4) {
      float kv[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int j = min(j0 + q * 64 + lane, sh.K - 1);
        float k, sy, sxx;
        if (j0 == 0) {
          k = c0[q]; sy = y0[q]; sxx = x0[q];
        } else {
          const int sj = sup[j];
          k = cs.get(j); sy = pc[2 * sj]; sxx = pc[2 * sj + 1];
        }
        if (w > 0.f) {
          const float dy = py - sy, dx = px - sxx;
          k += w * expf(-(dy * dy + dx * dx) * inv_tau);
        }
        kv[q] = k;
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int j = j0 + q * 64 + lane;
        if (j < sh.K && kv[q] > best) { best = kv[q]; bj = j; }
      }
    }
    argmax_step<32>(best, bj);
    argmax_step<16>(best, bj);
    argmax_step<8>(best, bj);
    argmax_step<4>(best, bj);
    argmax_step<2>(best, bj);
    argmax_step<1>(best, bj);
    pi_i = sup[(bj >= 0 && bj < sh.K) ? bj : 0];
  }
  if (lane == 0) {
    ws.pi[p * ws.s_pi + i] = pi_i;
    if (trace_assign) trace_assign[static_cast<long long>(p) * sh.N + i] = pi_i;
  }
}

template <typename T>
static hipError_t assign_impl(const Shape& sh, const Params& pr, const Ws& ws, const void* hidden_v,
                              bool support_ready, int32_t* trace_assign, hipStream_t st) {
  timer_mark(kStAssign, true, st);
  if (!support_ready) hipLaunchKernelGGL(support_kernel, dim3(sh.B), dim3(1024), 0, st, sh, ws);
  const int nblk = (sh.N + 3) / 4;
  if (sh.bounded) {
    const T* hidden = static_cast<const T*>(hidden_v);
    RowOperand<T> A{hidden, sh.d, static_cast<long long>(sh.N) * sh.d, nullptr, 0, sh.N};
    RowOperand<T> S{hidden, sh.d, static_cast<long long>(sh.N) * sh.d, ws.sup, ws.s_sup, sh.K};
    CosEpi epi{ws, sh.ldK, pr.norm_eps};
    hipError_t err;
    // 128-row tiles on 32x32 MFMA once they alone fill the chip twice over
    const long long big_tiles = static_cast<long long>((sh.N + kBigTile - 1) / kBigTile) *
                                ((sh.K + kBigTile - 1) / kBigTile) * sh.B;
    if constexpr (sizeof(T) == 2) {
      if (big_tiles >= 512) err = launch_gemm_nt_big(A, S, sh.d, sh.B, epi, st);
      else err = launch_gemm_nt<T, 64, 64>(A, S, sh.d, sh.B, epi, st);
    } else {
      err = launch_gemm_nt<T, 64, 64>(A, S, sh.d, sh.B, epi, st);
    }
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(gap_kernel<false>, dim3(nblk, sh.B), dim3(256), 0, st, sh, pr, ws);
  } else {
    hipLaunchKernelGGL(gap_kernel<true>, dim3(nblk, sh.B), dim3(256), 0, st, sh, pr, ws);
  }
  if (sh.bounded)
    hipLaunchKernelGGL(kappa_kernel<false>, dim3(nblk, sh.B), dim3(256), 0, st, sh, pr, ws, trace_assign);
  else
    hipLaunchKernelGGL(kappa_kernel<true>, dim3(nblk, sh.B), dim3(256), 0, st, sh, pr, ws, trace_assign);
  timer_mark(kStAssign, false, st);
  return hipGetLastError();
}

hipError_t launch_assignment(const Shape& sh, const Params& pr, const Ws& ws, const void* hidden,
                             bool support_ready, int32_t* trace_assign, hipStream_t st) {
  if (sh.dtype == 0) return assign_impl<float>(sh, pr, ws, hidden, support_ready, trace_assign, st);
  return assign_impl<bf16_t>(sh, pr, ws, hidden, support_ready, trace_assign, st);
}

}  // namespace gmc
