// Multi-image prompts (Sec. 3.1 totality rule; App. H "Batched complementary
// support"): the per-token image ids the image-restricted banks and the
// assignment read, and the seed set S_0 of one largest-singleton-gain token
// per image that the batched rounds start from.
#include "gmc_device.h"
#include "gmc_internal.h"
#include "gmc_kernels.h"

namespace gmc {

// One block per problem: ids clamped into [0, nimg), copied to the
// workspace, tokens counted per image; an id out of range or an image
// without tokens raises the input status bit.
__global__ void __launch_bounds__(1024) image_prep_kernel(Shape sh, Ws ws, const int32_t* image_id) {
  __shared__ int cnt[kMaxImages];
  __shared__ int bad;
  const int p = blockIdx.x, tid = threadIdx.x;
  if (tid < kMaxImages) cnt[tid] = 0;
  if (tid == 0) bad = 0;
  __syncthreads();
  const int32_t* src = image_id + static_cast<long long>(p) * sh.N;
  int* img = ws.img + p * ws.s_img;
  bool oob = false;
  for (int i = tid; i < sh.N; i += blockDim.x) {
    const int g = src[i];
    oob |= g < 0 || g >= sh.nimg;
    const int gc = min(max(g, 0), sh.nimg - 1);
    // written through like the row norms: the bank stream's kernels read
    // the ids after the row-norm gate, with no kernel boundary between
    __hip_atomic_store(&img[i], gc, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    atomicAdd(&cnt[gc], 1);
  }
  if (oob) atomicOr(&bad, 1);
  __syncthreads();
  if (tid < sh.nimg) {
    ws.imgcnt[p * ws.s_imgcnt + tid] = cnt[tid];
    if (cnt[tid] == 0) atomicOr(&bad, 1);
  }
  __syncthreads();
  if (tid == 0 && bad) raise_status(ws.cnt + p * ws.s_cnt, kStatusInput);
}

hipError_t launch_image_prep(const Shape& sh, const Ws& ws, const int32_t* image_id, hipStream_t st) {
  hipLaunchKernelGGL(image_prep_kernel, dim3(sh.B), dim3(1024), 0, st, sh, ws, image_id);
  return hipGetLastError();
}

// Singleton gains from the empty set, u_i = F({i}) = sum_m Cbar_mi: one wave
// per token over its contiguous client row.
__global__ void __launch_bounds__(256) seed_gain_kernel(Shape sh, Ws ws) {
  const int p = blockIdx.y, lane = threadIdx.x & 63;
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= sh.N) return;
  const float* alpha = ws.alpha + p * ws.s_m;
  const float* row = ws.E + p * ws.s_E + static_cast<long long>(i) * sh.ldM;
  float acc = 0.f;
  for (int m = lane * 4; m < sh.m; m += 256) {
    const float4 a = *reinterpret_cast<const float4*>(alpha + m);
    const float4 v = *reinterpret_cast<const float4*>(row + m);
    acc += fmaxf(a.x * v.x, 0.f);   // Cbar >= 0; also keeps padding columns inert
    acc += fmaxf(a.y * v.y, 0.f);
    acc += fmaxf(a.z * v.z, 0.f);
    acc += fmaxf(a.w * v.w, 0.f);
  }
  acc = wave_sum(acc);
  if (lane == 0) ws.u[p * ws.s_u + i] = acc;
}

// One block per problem: each image's seed is the token with the largest
// gain, ties to the lower index (packed keys: gain bits high, complemented
// index low, reduced with LDS maximum); it is marked selected (round 0),
// recorded at position g of the support order, and the coverage b_m(S_0)
// is stored for the rounds.  An image without tokens takes the lowest
// unselected token, so the support stays K distinct tokens.
__global__ void __launch_bounds__(1024) seed_pick_kernel(Shape sh, Ws ws) {
  __shared__ unsigned long long best[kMaxImages];
  __shared__ int seed[kMaxImages];
  const int p = blockIdx.x, tid = threadIdx.x;
  if (tid < kMaxImages) best[tid] = 0ull;
  __syncthreads();
  const float* u = ws.u + p * ws.s_u;
  const int* img = ws.img + p * ws.s_img;
  for (int i = tid; i < sh.N; i += blockDim.x) {
    const unsigned long long key = (static_cast<unsigned long long>(__float_as_uint(fmaxf(u[i], 0.f))) << 32) |
                                   static_cast<unsigned long long>(0xFFFFFFFFu - static_cast<unsigned>(i));
    atomicMax(&best[img[i]], key);
  }
  __syncthreads();
  int* sel = ws.sel + p * ws.s_sel;
  int* order = ws.order + p * ws.s_ord;
  if (tid == 0) {
    for (int g = 0; g < sh.nimg; ++g) {
      if (best[g] == 0ull) continue;
      const int i = static_cast<int>(0xFFFFFFFFu - static_cast<unsigned>(best[g] & 0xFFFFFFFFull));
      seed[g] = i;
      sel[i] = 0;
    }
    int next = 0;
    for (int g = 0; g < sh.nimg; ++g) {
      if (best[g] != 0ull) continue;
      while (next < sh.N && sel[next] >= 0) ++next;
      const int i = min(next, sh.N - 1);
      seed[g] = i;
      sel[i] = 0;
    }
    for (int g = 0; g < sh.nimg; ++g) order[g] = seed[g];
  }
  __syncthreads();
  const float* alpha = ws.alpha + p * ws.s_m;
  const float* E = ws.E + p * ws.s_E;
  float* cov = ws.cov + p * ws.s_cov;
  for (int m = tid; m < sh.m; m += blockDim.x) {
    const float a = alpha[m];
    float b = 0.f;
    for (int g = 0; g < sh.nimg; ++g) b = fmaxf(b, a * E[static_cast<long long>(seed[g]) * sh.ldM + m]);
    cov[m] = b;
  }
}

hipError_t launch_image_seeds(const Shape& sh, const Ws& ws, hipStream_t st) {
  hipLaunchKernelGGL(seed_gain_kernel, dim3((sh.N + 3) / 4, sh.B), dim3(256), 0, st, sh, ws);
  hipLaunchKernelGGL(seed_pick_kernel, dim3(sh.B), dim3(1024), 0, st, sh, ws);
  return hipGetLastError();
}

}  // namespace gmc
