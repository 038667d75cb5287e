// Signed-message realisation audit (App. G Eq. cond-message-error; App. I
// Eq. cond-message-decomposition, Eq. cond-softmax-bound, Eq.
// cond-message-polar; Prop. 2 Eq. message-bound).
//
// For every query/head client g = (h, t) the native attention of the next
// block is re-run twice, over the Full visual keys and values and over the
// compact ones at the K carriers, with the same nonvisual denominator:
//   y_g  = sum_i a_gi v_i,     y~_g = sum_j abar_gj v~_j,
//   M_gj = sum_(i in C_j) a_gi (the Full attention grouped by carrier),
//   term1_g = y_g - sum_j M_gj v~_j,  term2_g = sum_j (M_gj - abar_gj) v~_j,
//   l1_g = ||M_g - abar_g||_1,  bound_g = max_j |log M_gj + LSE_F - s~_gj|.
// Kernels: the Full pass (log-sum-exp, then attention written to scratch and
// the message), the carrier member lists, the grouped mass, the compact pass
// with every per-client statistic, and the weighted per-problem reduction
// (e_M, amplitude ratio, cosine).  fp32 throughout; one block per 16 clients
// of one kv head, keys and values staged through LDS in 64-row chunks.
#include "gmc_device.h"
#include "gmc_internal.h"
#include "gmc_kernels.h"

namespace gmc {

constexpr int kAudRows = 16;   // clients per block
constexpr int kAudChunk = 64;  // keys / values per LDS chunk

// Loads rows [c0, c0 + 64) of a [rows][Hkv][dh] tensor's kv head g into
// LDS as fp32 (pitch dh + 1), zero past `rows`.
template <typename T>
__device__ __forceinline__ void aud_stage(float* dst, const T* src, int c0, int rows, int g, int hkv, int dh) {
  const int pitch = dh + 1;
  for (int x = threadIdx.x; x < kAudChunk * dh; x += blockDim.x) {
    const int c = x / dh, d = x % dh;
    const int row = c0 + c;
    dst[c * pitch + d] = row < rows ? to_f32(src[(static_cast<long long>(row) * hkv + g) * dh + d]) : 0.f;
  }
}

// Client rows of block tile: r < 16 -> (h, t) of kv head g, or invalid.
struct AudTile {
  int p, g, rb, rows_g;
  __device__ AudTile(const Shape& sh) {
    p = blockIdx.z;
    g = blockIdx.y;
    rb = blockIdx.x * kAudRows;
    rows_g = sh.hg * sh.T;
  }
  __device__ bool valid(int r) const { return rb + r < rows_g; }
  __device__ int head(const Shape& sh, int r) const { return g * sh.hg + (rb + r) / sh.T; }
  __device__ int query(const Shape& sh, int r) const { return (rb + r) % sh.T; }
  // client row index m = h T + t of the problem
  __device__ int mrow(const Shape& sh, int r) const { return head(sh, r) * sh.T + query(sh, r); }
};

template <typename T>
__global__ void __launch_bounds__(256) audit_full_kernel(Shape sh, AudWs aw, const T* text_q, const T* vis_k,
                                                         const T* vis_v, const float* nonvis_lse) {
  extern __shared__ float lds[];
  const int dh = sh.dh, pitch = dh + 1, mg1 = sh.mg1;
  float* qs = lds;                                   // [16][pitch]
  float* ks = qs + kAudRows * pitch;                 // [64][pitch]
  float* as = ks + kAudChunk * pitch;                // [16][64]
  __shared__ float red_m[kAudRows][16], red_s[kAudRows][16], lse_s[kAudRows];
  const AudTile tl(sh);
  const int tid = threadIdx.x, r = tid >> 4, lc = tid & 15;
  const float scale = rsqrtf(static_cast<float>(dh));
  for (int x = tid; x < kAudRows * dh; x += blockDim.x) {
    const int rr = x / dh, d = x % dh;
    qs[rr * pitch + d] = tl.valid(rr) ? to_f32(text_q[((static_cast<long long>(tl.p) * sh.T + tl.query(sh, rr)) *
                                                       sh.hq + tl.head(sh, rr)) * dh + d]) : 0.f;
  }
  const T* kb = vis_k + static_cast<long long>(tl.p) * sh.N * sh.hkv * dh;
  const T* vb = vis_v + static_cast<long long>(tl.p) * sh.N * sh.hkv * dh;
  // pass 1: online max / sum of exp per client row (lane lc takes columns
  // lc, lc + 16, ... of each chunk)
  float mx = -INFINITY, sm = 0.f;
  for (int c0 = 0; c0 < sh.N; c0 += kAudChunk) {
    __syncthreads();
    aud_stage(ks, kb, c0, sh.N, tl.g, sh.hkv, dh);
    __syncthreads();
    for (int j = 0; j < kAudChunk / 16; ++j) {
      const int c = lc + 16 * j;
      if (c0 + c >= sh.N) continue;
      float s = 0.f;
      for (int d = 0; d < dh; ++d) s += qs[r * pitch + d] * ks[c * pitch + d];
      s *= scale;
      const float nm = fmaxf(mx, s);
      sm = sm * __expf(mx - nm) + __expf(s - nm);
      mx = nm;
    }
  }
  red_m[r][lc] = mx;
  red_s[r][lc] = sm;
  __syncthreads();
  if (tid < kAudRows) {
    float m = -INFINITY;
    for (int q = 0; q < 16; ++q) m = fmaxf(m, red_m[tid][q]);
    float s = 0.f;
    for (int q = 0; q < 16; ++q) s += red_m[tid][q] == -INFINITY ? 0.f : red_s[tid][q] * __expf(red_m[tid][q] - m);
    float D = m + logf(s);
    if (nonvis_lse && tl.valid(tid)) {
      const float nv = nonvis_lse[(static_cast<long long>(tl.p) * sh.hq + tl.head(sh, tid)) * sh.T + tl.query(sh, tid)];
      const float hi = fmaxf(D, nv), lo = fminf(D, nv);
      D = hi + log1pf(expf(lo - hi));
    }
    lse_s[tid] = D;
    if (tl.valid(tid)) aw.lse[static_cast<long long>(tl.p) * mg1 + tl.mrow(sh, tid)] = D;
  }
  __syncthreads();
  // pass 2: attention to scratch, message y_g = sum_i a_gi v_i (lane lc
  // takes dims lc, lc + 16, ...)
  const float D = lse_s[r];
  const bool rv = tl.valid(r);
  const int m = rv ? tl.mrow(sh, r) : 0;
  float y[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) y[k] = 0.f;
  float* A = aw.A + static_cast<long long>(tl.p) * sh.N * mg1;
  for (int c0 = 0; c0 < sh.N; c0 += kAudChunk) {
    __syncthreads();
    aud_stage(ks, kb, c0, sh.N, tl.g, sh.hkv, dh);
    __syncthreads();
    for (int j = 0; j < kAudChunk / 16; ++j) {
      const int c = lc + 16 * j;
      float a = 0.f;
      if (c0 + c < sh.N) {
        float s = 0.f;
        for (int d = 0; d < dh; ++d) s += qs[r * pitch + d] * ks[c * pitch + d];
        a = __expf(s * scale - D);
        if (rv) A[static_cast<long long>(c0 + c) * mg1 + m] = a;
      }
      as[r * kAudChunk + c] = a;
    }
    __syncthreads();
    aud_stage(ks, vb, c0, sh.N, tl.g, sh.hkv, dh);   // the values replace the keys
    __syncthreads();
    for (int c = 0; c < kAudChunk; ++c) {
      const float a = as[r * kAudChunk + c];
#pragma unroll
      for (int k = 0; k < 16; ++k)
        if (lc + 16 * k < dh) y[k] += a * ks[c * pitch + lc + 16 * k];
    }
  }
  if (rv) {
    float* yo = aw.Y + (static_cast<long long>(tl.p) * mg1 + m) * dh;
#pragma unroll
    for (int k = 0; k < 16; ++k)
      if (lc + 16 * k < dh) yo[lc + 16 * k] = y[k];
  }
}

// Carrier member lists (one thread per problem walks the tokens in order, so
// members are ascending within each carrier; slots are clamped to [0, K)).
__global__ void audit_members_kernel(Shape sh, AudWs aw, const int32_t* carrier) {
  const int p = blockIdx.x;
  if (threadIdx.x != 0) return;
  const int32_t* cr = carrier + static_cast<long long>(p) * sh.N;
  int* off = aw.off + static_cast<long long>(p) * (sh.K + 1);
  int* cur = aw.cur + static_cast<long long>(p) * sh.K;
  int* mem = aw.mem + static_cast<long long>(p) * sh.N;
  for (int j = 0; j <= sh.K; ++j) off[j] = 0;
  for (int i = 0; i < sh.N; ++i) off[min(max(cr[i], 0), sh.K - 1) + 1] += 1;
  for (int j = 0; j < sh.K; ++j) {
    off[j + 1] += off[j];
    cur[j] = off[j];
  }
  for (int i = 0; i < sh.N; ++i) mem[cur[min(max(cr[i], 0), sh.K - 1)]++] = i;
}

// Grouped Full mass M_gj = sum_(i in C_j) a_gi: one thread per client row,
// carriers in order, members in ascending order (coalesced over rows).
__global__ void __launch_bounds__(256) audit_mass_kernel(Shape sh, AudWs aw) {
  const int p = blockIdx.y, m = blockIdx.x * 256 + threadIdx.x;
  if (m >= sh.mg1) return;
  const int mg1 = sh.mg1;
  const int* off = aw.off + static_cast<long long>(p) * (sh.K + 1);
  const int* mem = aw.mem + static_cast<long long>(p) * sh.N;
  const float* A = aw.A + static_cast<long long>(p) * sh.N * mg1;
  float* Mt = aw.Mt + static_cast<long long>(p) * sh.K * mg1;
  for (int j = 0; j < sh.K; ++j) {
    float s = 0.f;
    for (int x = off[j]; x < off[j + 1]; ++x) s += A[static_cast<long long>(mem[x]) * mg1 + m];
    Mt[static_cast<long long>(j) * mg1 + m] = s;
  }
}

// Compact pass: abar over the carriers' keys (+ the same nonvisual part),
// y~, sum_j M_gj v~_j, the two decomposition terms, l1 and its bound, and
// every per-client statistic.
template <typename T>
__global__ void __launch_bounds__(256) audit_compact_kernel(Shape sh, AudWs aw, const T* text_q, const T* comp_k,
                                                            const T* comp_v, const float* nonvis_lse, float* rows_out,
                                                            float* vec_out) {
  extern __shared__ float lds[];
  const int dh = sh.dh, pitch = dh + 1, mg1 = sh.mg1;
  float* qs = lds;
  float* ks = qs + kAudRows * pitch;
  float* as = ks + kAudChunk * pitch;              // [16][64] abar
  float* ms = as + kAudRows * kAudChunk;           // [16][64] M
  __shared__ float red_m[kAudRows][16], red_s[kAudRows][16], lse_s[kAudRows];
  __shared__ float st[kAudRows][16][kAuditRow];
  const AudTile tl(sh);
  const int tid = threadIdx.x, r = tid >> 4, lc = tid & 15;
  const float scale = rsqrtf(static_cast<float>(dh));
  for (int x = tid; x < kAudRows * dh; x += blockDim.x) {
    const int rr = x / dh, d = x % dh;
    qs[rr * pitch + d] = tl.valid(rr) ? to_f32(text_q[((static_cast<long long>(tl.p) * sh.T + tl.query(sh, rr)) *
                                                       sh.hq + tl.head(sh, rr)) * dh + d]) : 0.f;
  }
  const T* kb = comp_k + static_cast<long long>(tl.p) * sh.K * sh.hkv * dh;
  const T* vb = comp_v + static_cast<long long>(tl.p) * sh.K * sh.hkv * dh;
  float mx = -INFINITY, sm = 0.f;
  for (int c0 = 0; c0 < sh.K; c0 += kAudChunk) {
    __syncthreads();
    aud_stage(ks, kb, c0, sh.K, tl.g, sh.hkv, dh);
    __syncthreads();
    for (int j = 0; j < kAudChunk / 16; ++j) {
      const int c = lc + 16 * j;
      if (c0 + c >= sh.K) continue;
      float s = 0.f;
      for (int d = 0; d < dh; ++d) s += qs[r * pitch + d] * ks[c * pitch + d];
      s *= scale;
      const float nm = fmaxf(mx, s);
      sm = sm * __expf(mx - nm) + __expf(s - nm);
      mx = nm;
    }
  }
  red_m[r][lc] = mx;
  red_s[r][lc] = sm;
  __syncthreads();
  if (tid < kAudRows) {
    float m = -INFINITY;
    for (int q = 0; q < 16; ++q) m = fmaxf(m, red_m[tid][q]);
    float s = 0.f;
    for (int q = 0; q < 16; ++q) s += red_m[tid][q] == -INFINITY ? 0.f : red_s[tid][q] * __expf(red_m[tid][q] - m);
    float D = m + logf(s);
    if (nonvis_lse && tl.valid(tid)) {
      const float nv = nonvis_lse[(static_cast<long long>(tl.p) * sh.hq + tl.head(sh, tid)) * sh.T + tl.query(sh, tid)];
      const float hi = fmaxf(D, nv), lo = fminf(D, nv);
      D = hi + log1pf(expf(lo - hi));
    }
    lse_s[tid] = D;
  }
  __syncthreads();
  const float D = lse_s[r];
  const bool rv = tl.valid(r);
  const int m = rv ? tl.mrow(sh, r) : 0;
  const float lse_f = rv ? aw.lse[static_cast<long long>(tl.p) * mg1 + m] : 0.f;
  const float* Mt = aw.Mt + static_cast<long long>(tl.p) * sh.K * mg1;
  float yc[16], my[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) { yc[k] = 0.f; my[k] = 0.f; }
  float l1 = 0.f, bound = 0.f;
  for (int c0 = 0; c0 < sh.K; c0 += kAudChunk) {
    __syncthreads();
    aud_stage(ks, kb, c0, sh.K, tl.g, sh.hkv, dh);
    __syncthreads();
    for (int j = 0; j < kAudChunk / 16; ++j) {
      const int c = lc + 16 * j;
      float a = 0.f, mm = 0.f;
      if (c0 + c < sh.K) {
        float s = 0.f;
        for (int d = 0; d < dh; ++d) s += qs[r * pitch + d] * ks[c * pitch + d];
        s *= scale;
        a = __expf(s - D);
        if (rv) {
          mm = Mt[static_cast<long long>(c0 + c) * mg1 + m];
          l1 += fabsf(mm - a);
          bound = fmaxf(bound, fabsf(logf(mm) + lse_f - s));
        }
      }
      as[r * kAudChunk + c] = a;
      ms[r * kAudChunk + c] = mm;
    }
    __syncthreads();
    aud_stage(ks, vb, c0, sh.K, tl.g, sh.hkv, dh);
    __syncthreads();
    for (int c = 0; c < kAudChunk; ++c) {
      const float a = as[r * kAudChunk + c], mm = ms[r * kAudChunk + c];
#pragma unroll
      for (int k = 0; k < 16; ++k)
        if (lc + 16 * k < dh) {
          const float v = ks[c * pitch + lc + 16 * k];
          yc[k] += a * v;
          my[k] += mm * v;
        }
    }
  }
  // per-client statistics: lane partials over its dims, then the 16 lanes
  const float* yf = aw.Y + (static_cast<long long>(tl.p) * mg1 + m) * dh;
  float acc[kAuditRow] = {};
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int d = lc + 16 * k;
    if (d >= dh || !rv) continue;
    const float y = yf[d], t1 = y - my[k], t2 = my[k] - yc[k], df = y - yc[k];
    acc[0] += y * y;
    acc[1] += yc[k] * yc[k];
    acc[2] += y * yc[k];
    acc[3] += df * df;
    acc[4] += t1 * t1;
    acc[5] += t2 * t2;
    if (vec_out) {
      float* vo = vec_out + ((static_cast<long long>(tl.p) * mg1 + m) * 4) * dh;
      vo[d] = y;
      vo[dh + d] = yc[k];
      vo[2 * dh + d] = t1;
      vo[3 * dh + d] = t2;
    }
  }
  acc[6] = l1;
  acc[7] = bound;
#pragma unroll
  for (int q = 0; q < kAuditRow; ++q) st[r][lc][q] = acc[q];
  __syncthreads();
  if (tid < kAudRows * kAuditRow) {
    const int rr = tid / kAuditRow, q = tid % kAuditRow;
    if (tl.valid(rr)) {
      float v = 0.f;
      for (int l = 0; l < 16; ++l) v = q == 7 ? fmaxf(v, st[rr][l][q]) : v + st[rr][l][q];
      const long long o = (static_cast<long long>(tl.p) * mg1 + tl.mrow(sh, rr)) * kAuditRow + q;
      aw.rowst[o] = v;
      if (rows_out) rows_out[o] = v;
    }
  }
}

// Weighted stack over the clients of a problem (sqrt(w_g) y_g): e_M, alpha,
// kappa and the norms; weights NULL = uniform 1 / (Hq T).
__global__ void __launch_bounds__(256) audit_reduce_kernel(Shape sh, AudWs aw, const float* weights, float* out) {
  __shared__ float red[16];
  const int p = blockIdx.x;
  float s[4] = {0.f, 0.f, 0.f, 0.f};
  float gap = -INFINITY;
  for (int m = threadIdx.x; m < sh.mg1; m += blockDim.x) {
    const int h = m / sh.T, t = m % sh.T;
    const float w = weights ? weights[(static_cast<long long>(p) * sh.hq + h) * sh.T + t] : 1.f / sh.mg1;
    const float* rs = aw.rowst + (static_cast<long long>(p) * sh.mg1 + m) * kAuditRow;
    s[0] += w * rs[0];
    s[1] += w * rs[1];
    s[2] += w * rs[2];
    s[3] += w * rs[3];
    gap = fmaxf(gap, rs[6] - rs[7]);
  }
  const float yy = block_sum(s[0], red), cc = block_sum(s[1], red);
  const float yc = block_sum(s[2], red), dd = block_sum(s[3], red);
  const float gmax = block_max(gap, red);
  if (threadIdx.x == 0) {
    float* o = out + static_cast<long long>(p) * kAuditOut;
    const float ny = sqrtf(yy), nc = sqrtf(cc), nd = sqrtf(dd);
    o[0] = nd / (ny + 1e-8f);
    o[1] = ny > 0.f ? nc / ny : 0.f;
    o[2] = (ny > 0.f && nc > 0.f) ? yc / (ny * nc) : 0.f;
    o[3] = ny;
    o[4] = nc;
    o[5] = nd;
    o[6] = gmax;
    o[7] = 0.f;
  }
}

// Dynamic LDS above 64 KB (head dimensions above 128) is granted once per kernel.
static hipError_t aud_lds(const void* fn, size_t bytes, int* granted) {
  if (bytes <= 64 * 1024 || static_cast<int>(bytes) <= *granted) return hipSuccess;
  const hipError_t err = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(bytes));
  if (err == hipSuccess) *granted = static_cast<int>(bytes);
  return err;
}

hipError_t launch_audit(const Shape& sh, const AudWs& aw, const void* text_q, const void* vis_k,
                        const void* vis_v, const void* comp_k, const void* comp_v, const int32_t* carrier,
                        const float* weights, const float* nonvis_lse, float* rows_out, float* vec_out, float* out,
                        hipStream_t st) {
  static int granted[4] = {0, 0, 0, 0};
  const int pitch = sh.dh + 1;
  const size_t lds_full = static_cast<size_t>(kAudRows + kAudChunk) * pitch * 4 + kAudRows * kAudChunk * 4;
  const size_t lds_comp = lds_full + kAudRows * kAudChunk * 4;
  const dim3 grid((sh.hg * sh.T + kAudRows - 1) / kAudRows, sh.hkv, sh.B);
  hipError_t err = sh.dtype == 0
                       ? aud_lds(reinterpret_cast<const void*>(audit_full_kernel<float>), lds_full, &granted[0])
                       : aud_lds(reinterpret_cast<const void*>(audit_full_kernel<bf16_t>), lds_full, &granted[1]);
  if (err == hipSuccess)
    err = sh.dtype == 0
              ? aud_lds(reinterpret_cast<const void*>(audit_compact_kernel<float>), lds_comp, &granted[2])
              : aud_lds(reinterpret_cast<const void*>(audit_compact_kernel<bf16_t>), lds_comp, &granted[3]);
  if (err != hipSuccess) return err;
  if (sh.dtype == 0) {
    hipLaunchKernelGGL(audit_full_kernel<float>, grid, dim3(256), lds_full, st, sh, aw,
                       static_cast<const float*>(text_q), static_cast<const float*>(vis_k),
                       static_cast<const float*>(vis_v), nonvis_lse);
  } else {
    hipLaunchKernelGGL(audit_full_kernel<bf16_t>, grid, dim3(256), lds_full, st, sh, aw,
                       static_cast<const bf16_t*>(text_q), static_cast<const bf16_t*>(vis_k),
                       static_cast<const bf16_t*>(vis_v), nonvis_lse);
  }
  hipLaunchKernelGGL(audit_members_kernel, dim3(sh.B), dim3(64), 0, st, sh, aw, carrier);
  hipLaunchKernelGGL(audit_mass_kernel, dim3((sh.mg1 + 255) / 256, sh.B), dim3(256), 0, st, sh, aw);
  if (sh.dtype == 0) {
    hipLaunchKernelGGL(audit_compact_kernel<float>, grid, dim3(256), lds_comp, st, sh, aw,
                       static_cast<const float*>(text_q), static_cast<const float*>(comp_k),
                       static_cast<const float*>(comp_v), nonvis_lse, rows_out, vec_out);
  } else {
    hipLaunchKernelGGL(audit_compact_kernel<bf16_t>, grid, dim3(256), lds_comp, st, sh, aw,
                       static_cast<const bf16_t*>(text_q), static_cast<const bf16_t*>(comp_k),
                       static_cast<const bf16_t*>(comp_v), nonvis_lse, rows_out, vec_out);
  }
  hipLaunchKernelGGL(audit_reduce_kernel, dim3(sh.B), dim3(256), 0, st, sh, aw, weights, out);
  return hipGetLastError();
}

}  // namespace gmc
