// LDS-staged MFMA GEMM for gfx950: C[p][r][c] = sum_k A[p][r][k] * B[p][c][k].
//
// Both operands are K-contiguous rows (the "NT" form every contraction of the
// operator takes: states x states, states x probe rows, projected states x
// projected states, states x selected states).  Rows may be gathered through
// an index list.  A block of 256 threads (4 waves, 2x2) computes a BM x BN
// tile; each wave owns (BM/2) x (BN/2) as 16x16 MFMA tiles.  K advances in
// steps of 32; the next global tile is prefetched into registers while the
// current LDS tile feeds the MFMAs.  The epilogue functor sees every valid
// output element and may also receive per-row sum/max over the block's
// columns (for the softmax-style bank normalisers).
#pragma once

#include "gmc_device.h"

namespace gmc {

template <typename T>
struct RowOperand {
  const T* base;      // element (p=0, row=0, k=0)
  long long ld;       // elements between consecutive rows
  long long pstride;  // elements between problems
  const int* gather;  // optional: row r reads source row gather[p*gstride + r]
  long long gstride;
  int rows;           // valid rows per problem
  __device__ __forceinline__ const T* row(int p, int r) const {
    long long src = gather ? static_cast<long long>(gather[p * gstride + r]) : r;
    return base + p * pstride + src * ld;
  }
};

constexpr int kGemmThreads = 256;
constexpr int kBK = 32;

template <typename T>
struct GemmSmem {
  // k-chunk pitch padded by 16 bytes to spread LDS banks between rows
  static constexpr int kPitch = kBK + 16 / static_cast<int>(sizeof(T));
};

// Epilogue contract:
//   __device__ void store(int p, int r, int c, float acc) const;
//   static constexpr bool kRowStats;
//   __device__ float value(int p, int r, int c, float acc) const;  // if kRowStats
//   __device__ void row_stats(int p, int r, int cblk, float sum, float mx) const;
template <typename T, int BM, int BN, class Epi>
__global__ void __launch_bounds__(kGemmThreads)
gemm_nt_kernel(RowOperand<T> A, RowOperand<T> B, int K, Epi epi) {
  constexpr int P = GemmSmem<T>::kPitch;
  constexpr int EPC = 16 / sizeof(T);                 // elements per 16-byte chunk
  constexpr int CPR = kBK / EPC;                      // chunks per tile row
  constexpr int A_CHUNKS = BM * CPR / kGemmThreads;   // per thread
  constexpr int B_CHUNKS = BN * CPR / kGemmThreads;
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int TM = WM / 16, TN = WN / 16;
  static_assert(A_CHUNKS >= 1 && B_CHUNKS >= 1, "tile too small");

  __shared__ __attribute__((aligned(16))) T As[BM * P];
  __shared__ __attribute__((aligned(16))) T Bs[BN * P];
  __shared__ float red_sum[2][BM];
  __shared__ float red_max[2][BM];

  const int p = blockIdx.z;
  const int row0 = blockIdx.y * BM, col0 = blockIdx.x * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;

  const T* a_src[A_CHUNKS];
  const T* b_src[B_CHUNKS];
#pragma unroll
  for (int i = 0; i < A_CHUNKS; ++i) {
    const int ch = tid + i * kGemmThreads, r = ch / CPR, kc = (ch % CPR) * EPC;
    a_src[i] = (row0 + r < A.rows) ? A.row(p, row0 + r) + kc : nullptr;
  }
#pragma unroll
  for (int i = 0; i < B_CHUNKS; ++i) {
    const int ch = tid + i * kGemmThreads, r = ch / CPR, kc = (ch % CPR) * EPC;
    b_src[i] = (col0 + r < B.rows) ? B.row(p, col0 + r) + kc : nullptr;
  }
  uint4 a_reg[A_CHUNKS], b_reg[B_CHUNKS];
  auto load_global = [&](int k0) {
#pragma unroll
    for (int i = 0; i < A_CHUNKS; ++i) a_reg[i] = a_src[i] ? ld16(a_src[i] + k0) : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < B_CHUNKS; ++i) b_reg[i] = b_src[i] ? ld16(b_src[i] + k0) : make_uint4(0, 0, 0, 0);
  };
  auto store_lds = [&]() {
#pragma unroll
    for (int i = 0; i < A_CHUNKS; ++i) {
      const int ch = tid + i * kGemmThreads, r = ch / CPR, kc = (ch % CPR) * EPC;
      st16(&As[r * P + kc], a_reg[i]);
    }
#pragma unroll
    for (int i = 0; i < B_CHUNKS; ++i) {
      const int ch = tid + i * kGemmThreads, r = ch / CPR, kc = (ch % CPR) * EPC;
      st16(&Bs[r * P + kc], b_reg[i]);
    }
  };

  floatx4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int nk = K / kBK;
  load_global(0);
  store_lds();
  __syncthreads();
  const int fr = lane & 15, fk = (lane >> 4) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) load_global((kt + 1) * kBK);
    Frag<T> fa[TM], fb[TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) fa[i] = frag_load<T>(&As[(wr * WM + i * 16 + fr) * P + fk]);
#pragma unroll
    for (int j = 0; j < TN; ++j) fb[j] = frag_load<T>(&Bs[(wc * WN + j * 16 + fr) * P + fk]);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = mma(fa[i], fb[j], acc[i][j]);
    __syncthreads();
    if (kt + 1 < nk) {
      store_lds();
      __syncthreads();
    }
  }

  // epilogue: lane holds column (lane&15), rows 4*(lane>>4)+e of each tile
  const int oc = lane & 15, orow = (lane >> 4) * 4;
  if constexpr (Epi::kRowStats) {
    float rs[TM][4], rm[TM][4];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) { rs[i][e] = 0.f; rm[i][e] = -INFINITY; }
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = row0 + wr * WM + i * 16 + orow + e;
          const int c = col0 + wc * WN + j * 16 + oc;
          if (r < A.rows && c < B.rows) {
            const float v = epi.value(p, r, c, acc[i][j][e]);
            rs[i][e] += v;
            rm[i][e] = fmaxf(rm[i][e], v);
          }
        }
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float s = group16_sum(rs[i][e]);
        const float m = group16_max(rm[i][e]);
        if (oc == 0) {
          const int rl = wr * WM + i * 16 + orow + e;
          red_sum[wc][rl] = s;
          red_max[wc][rl] = m;
        }
      }
    __syncthreads();
    for (int rl = tid; rl < BM; rl += kGemmThreads) {
      const int r = row0 + rl;
      if (r < A.rows)
        epi.row_stats(p, r, blockIdx.x, red_sum[0][rl] + red_sum[1][rl],
                      fmaxf(red_max[0][rl], red_max[1][rl]));
    }
  } else {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = row0 + wr * WM + i * 16 + orow + e;
          const int c = col0 + wc * WN + j * 16 + oc;
          if (r < A.rows && c < B.rows) epi.store(p, r, c, acc[i][j][e]);
        }
  }
}

template <typename T, int BM, int BN, class Epi>
inline hipError_t launch_gemm_nt(const RowOperand<T>& A, const RowOperand<T>& B, int K, int batch,
                                 const Epi& epi, hipStream_t stream) {
  dim3 grid((B.rows + BN - 1) / BN, (A.rows + BM - 1) / BM, batch);
  hipLaunchKernelGGL((gemm_nt_kernel<T, BM, BN, Epi>), grid, dim3(kGemmThreads), 0, stream, A, B, K,
                     epi);
  return hipGetLastError();
}

}  // namespace gmc
