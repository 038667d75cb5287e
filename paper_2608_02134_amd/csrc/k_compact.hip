// Sequence compaction after pruning (App. H "Index map and physical token
// accounting"; in the cached deployment the prompt K/V of the prefix layers
// is gathered at the retained sequence indices).
//
// A sequence of L positions holds its N visual tokens at [v0, v0 + N); K of
// them are retained (out_idx, ascending).  The compacted sequence has
// L2 = L - N + K positions and keeps every retained position in order, so
// both directions of the map are closed forms plus one binary search:
//   output j < v0           <- position j
//   v0 <= j < v0 + K        <- position v0 + out_idx[j - v0]
//   j >= v0 + K             <- position j + N - K
// and a visual position v0 + v maps to v0 + k where out_idx[k] = v, or to -1.
// Both kernels are pure data movement: 16-byte loads and stores, HBM-bound.
#include <algorithm>

#include "gmc_device.h"
#include "gmc_internal.h"
#include "gmc_kernels.h"

namespace gmc {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// One wave per position index x: the map of input position x (x < L) and
// output row x (x < L2) with its row and position ids.
__global__ void __launch_bounds__(256)
compact_sequence_kernel(int L, int v0, int N, int K, const int32_t* __restrict__ out_idx, int32_t* iota,
                        int32_t* keep, const uint4* __restrict__ seq_rows, const uint4* __restrict__ vis_rows,
                        uint4* out_rows, int row_chunks, const int32_t* __restrict__ seq_pos, int32_t* out_pos) {
  const int b = blockIdx.y, lane = threadIdx.x & 63;
  const int x = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int L2 = L - N + K;
  const int32_t* sel = out_idx + static_cast<long long>(b) * K;
  if (iota && x < L && lane == 0) {
    int m;
    if (x < v0) {
      m = x;
    } else if (x >= v0 + N) {
      m = x - (N - K);
    } else {
      // the retained rank of visual token x - v0 (binary search, ascending)
      const int v = x - v0;
      int lo = 0, hi = K;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (sel[mid] < v) lo = mid + 1; else hi = mid;
      }
      m = (lo < K && sel[lo] == v) ? v0 + lo : -1;
    }
    iota[static_cast<long long>(b) * L + x] = m;
  }
  if (x >= L2) return;
  const bool vis = x >= v0 && x < v0 + K;
  const int src = vis ? v0 + min(max(sel[x - v0], 0), N - 1) : (x < v0 ? x : x + N - K);
  if (keep && lane == 0) keep[static_cast<long long>(b) * L2 + x] = src;
  if (out_pos && lane < 3)
    out_pos[(static_cast<long long>(b) * L2 + x) * 3 + lane] = seq_pos[(static_cast<long long>(b) * L + src) * 3 + lane];
  if (out_rows) {
    const uint4* from = vis ? vis_rows + (static_cast<long long>(b) * K + (x - v0)) * row_chunks
                            : seq_rows + (static_cast<long long>(b) * L + src) * row_chunks;
    uint4* to = out_rows + (static_cast<long long>(b) * L2 + x) * row_chunks;
    for (int c = lane; c < row_chunks; c += 64) to[c] = from[c];   // (non-temporal measured slower here)
  }
}

// Up to kMaxGather tensors per launch, passed by value.
struct GatherTable {
  const uint4* src[kMaxGather];
  uint4* dst[kMaxGather];
};

// blockIdx.y = tensor; threads stride over the tensor's (sequence, row,
// 16-byte chunk) space, kGatherDepth chunks in flight per thread (32-bit
// indices: the host keeps a tensor below 2^31 chunks).  Every byte is moved
// once, so loads and stores are non-temporal (measured: 68% of HBM peak
// against 57% with cached ones).
constexpr int kGatherDepth = 4;
__global__ void __launch_bounds__(256)
gather_rows_kernel(GatherTable tab, int n_seq, int spk, int L, int L2, int row_chunks,
                   const int32_t* __restrict__ keep) {
  const uint4* src = tab.src[blockIdx.y];
  uint4* dst = tab.dst[blockIdx.y];
  const unsigned total = static_cast<unsigned>(n_seq) * L2 * row_chunks;
  const unsigned stride = gridDim.x * blockDim.x;
  const unsigned rc = row_chunks, l2 = L2;
  for (unsigned base = blockIdx.x * blockDim.x + threadIdx.x; base < total; base += kGatherDepth * stride) {
    u32x4 v[kGatherDepth];
    unsigned to[kGatherDepth];
#pragma unroll
    for (int u = 0; u < kGatherDepth; ++u) {
      const unsigned q = min(base + u * stride, total - 1);
      const unsigned r = q / rc;                 // s * L2 + j
      const unsigned c = q - r * rc;
      const unsigned s = r / l2;
      const unsigned j = r - s * l2;
      const int from = min(max(keep[static_cast<long long>(s / spk) * L2 + j], 0), L - 1);
      v[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src) +
                                        (static_cast<long long>(s) * L + from) * row_chunks + c);
      to[u] = q;
    }
#pragma unroll
    for (int u = 0; u < kGatherDepth; ++u)
      if (base + u * stride < total) __builtin_nontemporal_store(v[u], reinterpret_cast<u32x4*>(dst) + to[u]);
  }
}

hipError_t launch_compact_sequence(int B, int L, int v0, int N, int K, const int32_t* out_idx, int32_t* iota,
                                   int32_t* keep, const void* seq_rows, const void* vis_rows, void* out_rows,
                                   int row_chunks, const int32_t* seq_pos, int32_t* out_pos, hipStream_t st) {
  const int span = max(L, L - N + K);
  hipLaunchKernelGGL(compact_sequence_kernel, dim3((span + 3) / 4, B), dim3(256), 0, st, L, v0, N, K, out_idx, iota,
                     keep, static_cast<const uint4*>(seq_rows), static_cast<const uint4*>(vis_rows),
                     static_cast<uint4*>(out_rows), row_chunks, seq_pos, out_pos);
  return hipGetLastError();
}

hipError_t launch_gather_rows(int n_tensors, const void* const* src, void* const* dst, int n_seq, int spk, int L,
                              int L2, int row_chunks, const int32_t* keep, hipStream_t st) {
  GatherTable tab{};
  for (int t = 0; t < n_tensors; ++t) {
    tab.src[t] = static_cast<const uint4*>(src[t]);
    tab.dst[t] = static_cast<uint4*>(dst[t]);
  }
  const long long total = static_cast<long long>(n_seq) * L2 * row_chunks;
  // about eight resident blocks per CU over all tensors, kGatherDepth chunks
  // per thread and trip
  const long long want = (total + 1LL * kGatherDepth * 256 - 1) / (1LL * kGatherDepth * 256);
  const long long cap = std::max<long long>(1, 32768 / n_tensors);
  const int gx = static_cast<int>(std::max<long long>(1, std::min(want, cap)));
  hipLaunchKernelGGL(gather_rows_kernel, dim3(gx, n_tensors), dim3(256), 0, st, tab, n_seq, spk, L, L2, row_chunks,
                     keep);
  return hipGetLastError();
}

}  // namespace gmc
