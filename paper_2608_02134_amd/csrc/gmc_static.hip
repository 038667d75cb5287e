// gmc_prune_static: the operator without any device allocation.  Its
// workspace is carved out of a file-scope device array of fixed size instead
// of the context's allocation, so a caller that cannot allocate device memory
// (code under graph capture, tight serving loops, harnesses that forbid
// allocation) can still prune.  The array's device address is looked up once
// per device, on the entry point's first call there; host code uses only that
// address (the array's name is a host-side stand-in).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>

#include "gmc.h"
#include "gmc_internal.h"
#include "gmc_kernels.h"
#include "gmc_path.h"

namespace {

constexpr size_t kScratchBytes = GMC_STATIC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

// One copy per device, held until the process ends.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The call's workspace region starts cleared: earlier calls of another shape
// left their data at other offsets.
__global__ void __launch_bounds__(256) zero_fill_kernel(uint4* p, long long n16) {
  const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
  for (long long i = blockIdx.x * static_cast<long long>(blockDim.x) + threadIdx.x; i < n16; i += stride)
    p[i] = make_uint4(0u, 0u, 0u, 0u);
}

}  // namespace

extern "C" int gmc_prune_static(const gmc_config* cfg, int64_t B, const void* hidden, const void* text_q,
                                const void* vis_k, const int32_t* pos3d, int64_t N, int64_t T, int64_t K,
                                void* out_hidden, int32_t* out_pos, int32_t* out_idx, const float* nonvis_lse,
                                void* stream) {
  using namespace gmc;
  if (!cfg) return set_error(GMC_ERR_ARG, "gmc_prune_static: cfg is NULL");
  if (B < 1 || N < 1 || T < 0 || B > (1 << 20) || N > kMaxN || T > (1 << 20))
    return set_error(GMC_ERR_ARG, "gmc_prune_static: need B >= 1, 1 <= N <= %d, T >= 0 (B=%lld N=%lld T=%lld)",
                     kMaxN, static_cast<long long>(B), static_cast<long long>(N), static_cast<long long>(T));
  // the call's own shape is the workspace's capacity
  gmc_config c = *cfg;
  c.max_batch = static_cast<int32_t>(B);
  c.max_n = static_cast<int32_t>(N);
  c.max_t = static_cast<int32_t>(T);
  c.max_k = static_cast<int32_t>(gmc_realized_k(N, K));
  c.max_hist_views = 0;   // no historical views and one image on this entry point
  c.max_images = 1;
  int rc = check_config(&c);
  if (rc != GMC_OK) return rc;
  Shape s;
  rc = resolve_shape(c, Limits{c.max_batch, c.max_n, c.max_t, c.max_k, 0, 1}, B, N, T, K, &s);
  if (rc != GMC_OK) return rc;
  rc = check_tensors(s, hidden, text_q, vis_k, pos3d, out_hidden, out_pos, out_idx);
  if (rc != GMC_OK) return rc;
  Ws ws{};
  const size_t bytes = carve_workspace(c, nullptr, &ws);
  if (bytes > kScratchBytes)
    return set_error(GMC_ERR_CAPACITY,
                     "gmc_prune_static: this call needs %zu bytes of workspace; the static scratch holds %zu "
                     "(use gmc_init + gmc_prune)", bytes, kScratchBytes);
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return set_error(GMC_ERR_HIP, "gmc_prune_static: no HIP device (%s)", hipGetErrorString(err));
  if (dev < 0 || dev >= kMaxDevices) return set_error(GMC_ERR_HIP, "gmc_prune_static: device %d not supported", dev);
  void* base = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
      void* ptr = nullptr;
      err = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
      if (err != hipSuccess || !ptr)
        return set_error(GMC_ERR_HIP, "gmc_prune_static: device scratch address (%s)", hipGetErrorString(err));
      g_scratch_ptr[dev] = ptr;
    }
    base = g_scratch_ptr[dev];
  }
  carve_workspace(c, static_cast<char*>(base), &ws);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (s.K < s.N) {
    const long long n16 = static_cast<long long>(bytes / 16);
    const int blocks = static_cast<int>(std::min<long long>(1024, (n16 + 255) / 256));
    hipLaunchKernelGGL(zero_fill_kernel, dim3(std::max(blocks, 1)), dim3(256), 0, st, static_cast<uint4*>(base), n16);
    err = hipGetLastError();
    if (err != hipSuccess) return set_error(GMC_ERR_HIP, "gmc_prune_static: clearing the scratch (%s)",
                                            hipGetErrorString(err));
  }
  const Params pr = params_of(c);
  const PathStreams ps{st, nullptr, 0, nullptr, nullptr};
  bool cert = false;
  return enqueue_prune(c, pr, ws, s, ps, 0, hidden, text_q, vis_k, pos3d, out_hidden, out_pos, out_idx, nonvis_lse,
                       gmc_trace{}, &cert);
}
