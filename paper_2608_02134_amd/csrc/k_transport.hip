// Population transport and physical compaction (Sec. 3.4 Eq. transport; App.
// H Eq. cond-transport, Eq. cond-population-gate, and "Index map and physical
// token accounting").
//
// One block per support member j (slot order = ascending source index):
// members i with pi(i) = j are found by a ballot scan of pi in ascending
// order and accumulated as m_i h_i in fp32 registers in that fixed order
// (bitwise repeatable, no atomics).  Then c_j = acc / M_j, the blend
// (1 - tau_j) h_j + tau_j c_j, RMS restoration to rms(h_j), one cast to the
// residual dtype, and the compact write of the state, the original (t,h,w)
// ids and the source index.  HBM traffic is one read of every member row.
#include "gmc_device.h"
#include "gmc_internal.h"
#include "gmc_kernels.h"

namespace gmc {

template <typename T, int G>
__global__ void __launch_bounds__(256)
transport_kernel(Shape sh, Params pr, Ws ws, const T* hidden, const int32_t* pos3d, T* out_hidden,
                 int32_t* out_pos, int32_t* out_idx) {
  constexpr int CH = sizeof(T) == 2 ? 1 : 2;   // 16-byte chunks per 8-element group
  // member rows loaded together (about 128 registers of row data)
  constexpr int kMB = 128 / (G * CH * 4) < 1 ? 1 : (128 / (G * CH * 4) > 8 ? 8 : 128 / (G * CH * 4));
  constexpr int kPiQ = 8;                 // assignment entries per thread and pass
  __shared__ unsigned long long masks[kPiQ][4];
  __shared__ int members[kPiQ * 256];
  __shared__ float weights[kPiQ * 256];
  __shared__ float red[16];
  const int jj = blockIdx.x, p = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = wave_id();
  const unsigned long long below = (1ull << lane) - 1ull;
  const int j = ws.sup[p * ws.s_sup + jj];
  const int* pi = ws.pi + p * ws.s_pi;
  const float* eb = ws.ebar + p * ws.s_eb;
  const float sx = ws.gate[p * ws.s_gate];
  const float inv_mean = ws.gate[p * ws.s_gate + 2];   // 0: uniform fallback ebar = 1
  const float m0 = 1.f - pr.pop_strength * sx, m1 = pr.pop_strength * sx;
  const T* H = hidden + static_cast<long long>(p) * sh.N * sh.d;
  const int ngroups = sh.d / 8;
  // the carrier's own row and norm go out first (they need only j)
  const T* hj = H + static_cast<long long>(j) * sh.d;
  uint4 own[G][CH];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int grp = min(tid + g * 256, ngroups - 1);
#pragma unroll
    for (int c = 0; c < CH; ++c) own[g][c] = ld16(hj + grp * 8 + c * 4);
  }
  const float n2j = ws.n2[p * ws.s_n + j];
  float acc[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[g][e] = 0.f;
  float mass = 0.f;
  for (int base = 0; base < sh.N; base += kPiQ * 256) {
    // the ordered member list of this pass (ascending source index) with each
    // member's population weight m_i: the assignment and ebar loads of the
    // pass are all in flight together, one ballot per 256 tokens
    int pv[kPiQ];
    float ev[kPiQ];
#pragma unroll
    for (int q = 0; q < kPiQ; ++q) {
      const int i = base + q * 256 + tid;
      pv[q] = i < sh.N ? pi[i] : -1;
      ev[q] = i < sh.N ? eb[i] : 0.f;
    }
    unsigned long long bal[kPiQ];
#pragma unroll
    for (int q = 0; q < kPiQ; ++q) bal[q] = __ballot(pv[q] == j);
    __syncthreads();   // the previous pass is done with masks, members and weights
    if (lane == 0)
#pragma unroll
      for (int q = 0; q < kPiQ; ++q) masks[q][wave] = bal[q];
    __syncthreads();
    // offsets of the 4 * kPiQ ballot words (order q-major, then wave): lane
    // l < 32 of every wave counts word l, one wave scan gives the prefixes
    const int cnt = lane < 4 * kPiQ ? __popcll(masks[lane >> 2][lane & 3]) : 0;
    const int incl = wave_scan_add(cnt);
    const int total = __builtin_amdgcn_readlane(incl, 4 * kPiQ - 1);
#pragma unroll
    for (int q = 0; q < kPiQ; ++q) {
      const int w = q * 4 + wave;
      const int off = __builtin_amdgcn_readlane(incl - cnt, w);
      if ((bal[q] >> lane) & 1ull) {
        const int slot = off + __popcll(bal[q] & below);
        members[slot] = base + q * 256 + tid;
        weights[slot] = m0 + m1 * (inv_mean > 0.f ? ev[q] * inv_mean : 1.f);
      }
    }
    __syncthreads();
    for (int b0 = 0; b0 < total; b0 += kMB) {
      // every member row of the batch is requested before any accumulation;
      // slots past the list end repeat its last row with weight 0, which
      // leaves the fp32 sums bit-identical (finite rows) and keeps the
      // accumulation free of branches, so the loads are not sunk into them
      uint4 raw[kMB][G][CH];
#pragma unroll
      for (int q = 0; q < kMB; ++q) {
        const int ii = members[min(b0 + q, total - 1)];
        const T* row = H + static_cast<long long>(ii) * sh.d;
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const int grp = min(tid + g * 256, ngroups - 1);
#pragma unroll
          for (int c = 0; c < CH; ++c) raw[q][g][c] = ld16(row + grp * 8 + c * 4);
        }
      }
#pragma unroll
      for (int q = 0; q < kMB; ++q) {
        const float mi = b0 + q < total ? weights[b0 + q] : 0.f;
        mass += mi;
#pragma unroll
        for (int g = 0; g < G; ++g) {
          if constexpr (sizeof(T) == 2) {
            const bf16_t* v = reinterpret_cast<const bf16_t*>(&raw[q][g][0]);
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[g][e] += mi * bf16_to_f32(v[e]);
          } else {
            const float* v = reinterpret_cast<const float*>(&raw[q][g][0]);
            const float* v2 = reinterpret_cast<const float*>(&raw[q][g][1]);
#pragma unroll
            for (int e = 0; e < 4; ++e) { acc[g][e] += mi * v[e]; acc[g][e + 4] += mi * v2[e]; }
          }
        }
      }
    }
  }
  // blend with the carrier's own state and restore its RMS
  const float inv_mass = 1.f / mass;
  float ss = 0.f;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int grp = tid + g * 256;
    if (grp < ngroups) {
      float hv[8];
      if constexpr (sizeof(T) == 2) {
        const bf16_t* v = reinterpret_cast<const bf16_t*>(&own[g][0]);
#pragma unroll
        for (int e = 0; e < 8; ++e) hv[e] = bf16_to_f32(v[e]);
      } else {
        const float* v = reinterpret_cast<const float*>(&own[g][0]);
        const float* v2 = reinterpret_cast<const float*>(&own[g][1]);
#pragma unroll
        for (int e = 0; e < 4; ++e) { hv[e] = v[e]; hv[e + 4] = v2[e]; }
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float v = (1.f - pr.tau_j) * hv[e] + pr.tau_j * (acc[g][e] * inv_mass);
        acc[g][e] = v;
        ss += v * v;
      }
    }
  }
  ss = block_sum(ss, red);
  const float rms_v = sqrtf(ss / static_cast<float>(sh.d));
  const float rms_h = sqrtf(n2j / static_cast<float>(sh.d));
  const float scale = rms_h / (rms_v + pr.restore_eps);
  T* out = out_hidden + (static_cast<long long>(p) * sh.K + jj) * sh.d;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int grp = tid + g * 256;
    if (grp < ngroups) {
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = acc[g][e] * scale;
      store8_f32<T>(out + grp * 8, v);
    }
  }
  if (tid < 3) {
    out_pos[(static_cast<long long>(p) * sh.K + jj) * 3 + tid] =
        pos3d[(static_cast<long long>(p) * sh.N + j) * 3 + tid];
  }
  if (tid == 0) out_idx[static_cast<long long>(p) * sh.K + jj] = j;
}

template <typename T>
static hipError_t transport_impl(const Shape& sh, const Params& pr, const Ws& ws, const void* hidden,
                                 const int32_t* pos3d, void* out_hidden, int32_t* out_pos,
                                 int32_t* out_idx, hipStream_t st) {
  const dim3 grid(sh.K, sh.B);
  const int groups_per_thread = (sh.d / 8 + 255) / 256;
  const T* h = static_cast<const T*>(hidden);
  T* o = static_cast<T*>(out_hidden);
  timer_mark(kStTransport, true, st);
  if (groups_per_thread <= 1)
    hipLaunchKernelGGL((transport_kernel<T, 1>), grid, dim3(256), 0, st, sh, pr, ws, h, pos3d, o, out_pos, out_idx);
  else if (groups_per_thread <= 2)
    hipLaunchKernelGGL((transport_kernel<T, 2>), grid, dim3(256), 0, st, sh, pr, ws, h, pos3d, o, out_pos, out_idx);
  else if (groups_per_thread <= 4)
    hipLaunchKernelGGL((transport_kernel<T, 4>), grid, dim3(256), 0, st, sh, pr, ws, h, pos3d, o, out_pos, out_idx);
  else if (groups_per_thread <= 8)
    hipLaunchKernelGGL((transport_kernel<T, 8>), grid, dim3(256), 0, st, sh, pr, ws, h, pos3d, o, out_pos, out_idx);
  else
    return hipErrorInvalidValue;
  timer_mark(kStTransport, false, st);
  return hipGetLastError();
}

hipError_t launch_transport(const Shape& sh, const Params& pr, const Ws& ws, const void* hidden,
                            const int32_t* pos3d, void* out_hidden, int32_t* out_pos,
                            int32_t* out_idx, hipStream_t st) {
  if (sh.dtype == 0)
    return transport_impl<float>(sh, pr, ws, hidden, pos3d, out_hidden, out_pos, out_idx, st);
  return transport_impl<bf16_t>(sh, pr, ws, hidden, pos3d, out_hidden, out_pos, out_idx, st);
}

// ---------------------------------------------------------------------------
// K = N identity and debug exports
// ---------------------------------------------------------------------------
__global__ void iota_kernel(int32_t* out_idx, int n, int batch) {
  const long long total = static_cast<long long>(n) * batch;
  for (long long x = blockIdx.x * static_cast<long long>(blockDim.x) + threadIdx.x; x < total;
       x += static_cast<long long>(gridDim.x) * blockDim.x)
    out_idx[x] = static_cast<int32_t>(x % n);
}

hipError_t launch_identity(const Shape& sh, const void* hidden, const int32_t* pos3d,
                           void* out_hidden, int32_t* out_pos, int32_t* out_idx, hipStream_t st) {
  const size_t esz = sh.dtype == 0 ? 4 : 2;
  hipError_t err = hipMemcpyAsync(out_hidden, hidden, esz * sh.B * sh.N * sh.d, hipMemcpyDeviceToDevice, st);
  if (err != hipSuccess) return err;
  err = hipMemcpyAsync(out_pos, pos3d, sizeof(int32_t) * 3 * sh.B * sh.N, hipMemcpyDeviceToDevice, st);
  if (err != hipSuccess) return err;
  const long long total = static_cast<long long>(sh.B) * sh.N;
  const int blocks = static_cast<int>(min(4096LL, (total + 255) / 256));
  hipLaunchKernelGGL(iota_kernel, dim3(blocks), dim3(256), 0, st, out_idx, sh.N, sh.B);
  return hipGetLastError();
}

__global__ void export_client_kernel(Shape sh, Ws ws, float* out) {
  const int p = blockIdx.z, m = blockIdx.y;
  const float a = ws.alpha[p * ws.s_m + m];
  const float* E = ws.E + p * ws.s_E + m;
  float* o = out + (static_cast<long long>(p) * sh.m + m) * sh.N;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < sh.N; i += gridDim.x * blockDim.x)
    o[i] = a * E[static_cast<long long>(i) * sh.ldM];
}

// One wave per problem: the selection's statistics, the device status word
// (completion-counter slot 7) and the per-bank objectives F_b(S) = sum of the
// final coverage b_m and F_b(V) = sum of max_i Cbar_mi over the bank's rows
// (grounded, appearance, spatial), from which omega_b = F_b(V) / F(V) and the
// saturation c_b = F_b(S) / F_b(V) follow (Eq. cond-bank-mixture).
__global__ void export_stats_kernel(Shape sh, Ws ws, float* out) {
  const int p = blockIdx.x, t = threadIdx.x;
  float* o = out + p * kStats;
  if (t < 8) o[t] = ws.stats[p * ws.s_st + t];
  if (t == 8) o[8] = static_cast<float>(ws.cnt[p * ws.s_cnt + 7]);
  const float* cov = ws.cov + p * ws.s_cov;
  const float* peak = ws.peak + p * ws.s_m;
  const int lo[3] = {0, sh.mg, sh.mg + sh.mv}, hi[3] = {sh.mg, sh.mg + sh.mv, sh.m};
#pragma unroll
  for (int b = 0; b < 3; ++b) {
    float fs = 0.f, fv = 0.f;
    for (int m = lo[b] + t; m < hi[b]; m += 64) {
      fs += cov[m];
      fv += peak[m];
    }
    fs = wave_sum(fs);
    fv = wave_sum(fv);
    if (t == 0) {
      o[9 + b] = fs;
      o[12 + b] = fv;
    }
  }
}

__global__ void export_ebar_kernel(Shape sh, Ws ws, float* out) {
  const int p = blockIdx.y;
  const float inv_mean = ws.gate[p * ws.s_gate + 2];
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < sh.N; i += gridDim.x * blockDim.x)
    out[static_cast<long long>(p) * sh.N + i] = inv_mean > 0.f ? ws.ebar[p * ws.s_eb + i] * inv_mean : 1.f;
}

hipError_t launch_trace_exports(const Shape& sh, const Ws& ws, float* trace_client, float* trace_stats,
                                float* trace_ebar, hipStream_t st) {
  if (trace_ebar)
    hipLaunchKernelGGL(export_ebar_kernel, dim3((sh.N + 255) / 256, sh.B), dim3(256), 0, st, sh, ws, trace_ebar);
  if (trace_client)
    hipLaunchKernelGGL(export_client_kernel, dim3((sh.N + 255) / 256, sh.m, sh.B), dim3(256), 0, st, sh,
                       ws, trace_client);
  if (trace_stats) hipLaunchKernelGGL(export_stats_kernel, dim3(sh.B), dim3(64), 0, st, sh, ws, trace_stats);
  return hipGetLastError();
}

}  // namespace gmc
