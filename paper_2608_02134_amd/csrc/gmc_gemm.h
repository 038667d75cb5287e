// LDS-staged MFMA GEMM for gfx950: C[p][r][c] = sum_k A[p][r][k] * B[p][c][k].
//
// Both operands are K-contiguous rows (the "NT" form every contraction of the
// operator takes: states x states, states x probe rows, projected states x
// projected states, states x selected states).  Rows may be gathered through
// an index list.  A block of 256 threads (4 waves, 2x2) computes a BM x BN
// tile; each wave owns (BM/2) x (BN/2) as 16x16 MFMA tiles.  K advances in
// slabs of 64: global loads run kStages slabs ahead in register stages (so a
// slab's loads have kStages - 1 slabs of MFMA work to arrive), the LDS tile is
// double-buffered, one barrier per slab.  Row indices are
// clamped so every load is unconditional; out-of-range rows and columns are
// masked in the epilogue.  The epilogue functor gets a per-row and a
// per-column scale (loaded once per lane) and sees every valid element; it may
// also receive per-row sum/max over the block's columns.
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
constexpr int kBK = 64;
// register stages of the slab pipeline: eight 16-byte chunks per thread and
// stage cost 32 registers, so fp32 operands (twice the chunks) get half
template <typename T>
constexpr int gemm_stages() { return sizeof(T) == 2 ? 8 : 4; }

// Epilogue contract (p is the problem index, or problem * ksplit + split):
//   static constexpr bool kRowStats;
//   __device__ float row_scale(int p, int r) const;   // r valid
//   __device__ float col_scale(int p, int c) const;   // c valid
//   __device__ float value(int p, int r, int c, float acc_scaled) const;  // stores; returns value
//   __device__ void row_stats(int p, int r, int cblk, float sum, float mx) const;
template <typename T, int BM, int BN, class Epi>
__global__ void __launch_bounds__(kGemmThreads)
gemm_nt_kernel(RowOperand<T> A, RowOperand<T> B, int K, int ksplit, Epi epi) {
  constexpr int EPC = 16 / sizeof(T);                 // elements per 16-byte chunk
  constexpr int P = kBK + EPC;                        // LDS row pitch (elements), 16 B pad
  constexpr int CPR = kBK / EPC;                      // chunks per tile row
  constexpr int A_CHUNKS = BM * CPR / kGemmThreads;   // per thread per slab
  constexpr int B_CHUNKS = BN * CPR / kGemmThreads;
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int TM = WM / 16, TN = WN / 16;
  static_assert(A_CHUNKS >= 1 && B_CHUNKS >= 1, "tile too small");

  __shared__ __attribute__((aligned(16))) T As[2][BM * P];
  __shared__ __attribute__((aligned(16))) T Bs[2][BN * P];
  __shared__ float red_sum[2][BM];
  __shared__ float red_max[2][BM];

  // blockIdx.z = problem * ksplit + split: split s covers K columns
  // [s*K, (s+1)*K) (K is the per-split length); the epilogue sees the
  // combined index, so a split-K epilogue can keep its partial sums apart
  const int pe = blockIdx.z, p = pe / ksplit, ks0 = (pe % ksplit) * K;
  const int row0 = blockIdx.y * BM, col0 = blockIdx.x * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;

  const T* a_src[A_CHUNKS];
  const T* b_src[B_CHUNKS];
#pragma unroll
  for (int i = 0; i < A_CHUNKS; ++i) {
    const int ch = tid + i * kGemmThreads, r = ch / CPR, kc = (ch % CPR) * EPC;
    a_src[i] = A.row(p, min(row0 + r, A.rows - 1)) + ks0 + kc;
  }
#pragma unroll
  for (int i = 0; i < B_CHUNKS; ++i) {
    const int ch = tid + i * kGemmThreads, r = ch / CPR, kc = (ch % CPR) * EPC;
    b_src[i] = B.row(p, min(col0 + r, B.rows - 1)) + ks0 + kc;
  }
  constexpr int S = gemm_stages<T>();
  uint4 ra[S][A_CHUNKS], rb[S][B_CHUNKS];
  const int nk = K / kBK;
  auto load = [&](int kt, uint4* ra, uint4* rb) {
    const int k0 = min(kt, nk - 1) * kBK;
#pragma unroll
    for (int i = 0; i < A_CHUNKS; ++i) ra[i] = ld16(a_src[i] + k0);
#pragma unroll
    for (int i = 0; i < B_CHUNKS; ++i) rb[i] = ld16(b_src[i] + k0);
  };
  auto store = [&](int buf, const uint4* ra, const uint4* rb) {
#pragma unroll
    for (int i = 0; i < A_CHUNKS; ++i) {
      const int ch = tid + i * kGemmThreads, r = ch / CPR, kc = (ch % CPR) * EPC;
      st16(&As[buf][r * P + kc], ra[i]);
    }
#pragma unroll
    for (int i = 0; i < B_CHUNKS; ++i) {
      const int ch = tid + i * kGemmThreads, r = ch / CPR, kc = (ch % CPR) * EPC;
      st16(&Bs[buf][r * P + kc], rb[i]);
    }
  };

  floatx4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int fr = lane & 15, fk = (lane >> 4) * 8;
  auto compute = [&](int buf) {
#pragma unroll
    for (int ks = 0; ks < kBK; ks += 32) {
      Frag<T> fa[TM], fb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) fa[i] = frag_load<T>(&As[buf][(wr * WM + i * 16 + fr) * P + ks + fk]);
#pragma unroll
      for (int j = 0; j < TN; ++j) fb[j] = frag_load<T>(&Bs[buf][(wc * WN + j * 16 + fr) * P + ks + fk]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mma(fa[i], fb[j], acc[i][j]);
    }
  };

  // prologue: slabs 0..S-1 in flight, slab 0 in LDS buffer 0
#pragma unroll
  for (int s = 0; s < S; ++s) load(s, ra[s], rb[s]);
  store(0, ra[0], rb[0]);
  __syncthreads();
  // steady state, unrolled by S so the register stages are static: step s
  // computes slab kt+s from LDS buffer s&1, refills its now free stage with
  // slab kt+s+S and moves slab kt+s+1 into the other buffer (past the last
  // slab these are clamped copies, never read)
  // The main loop runs whole groups of S steps with no exit inside the
  // group, so every path into its head has the same loads in flight and the
  // compiler's wait counts stay exact (an exit inside the unrolled group
  // merges those paths and forces a wait for every load at the head).  The
  // last nk % S slabs are already loaded: the tail only computes and stores.
  const int nk_main = nk - nk % S;
  for (int kt = 0; kt < nk_main; kt += S) {
#pragma unroll
    for (int s = 0; s < S; ++s) {
      load(kt + s + S, ra[s], rb[s]);
      compute(s & 1);
      store((s + 1) & 1, ra[(s + 1) % S], rb[(s + 1) % S]);
      __syncthreads();
    }
  }
#pragma unroll
  for (int s = 0; s < S - 1; ++s) {
    if (nk_main + s >= nk) break;
    compute(s & 1);
    store((s + 1) & 1, ra[(s + 1) % S], rb[(s + 1) % S]);
    __syncthreads();
  }

  // epilogue: lane holds column (lane&15), rows 4*(lane>>4)+e of each tile
  const int oc = lane & 15, orow = (lane >> 4) * 4;
  float rsc[TM][4], csc[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e)
      rsc[i][e] = epi.row_scale(pe, min(row0 + wr * WM + i * 16 + orow + e, A.rows - 1));
#pragma unroll
  for (int j = 0; j < TN; ++j) csc[j] = epi.col_scale(pe, min(col0 + wc * WN + j * 16 + oc, B.rows - 1));

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
          const float v = epi.value(pe, r, c, acc[i][j][e] * rsc[i][e] * csc[j]);
          if constexpr (Epi::kRowStats) {
            rs[i][e] += v;
            rm[i][e] = fmaxf(rm[i][e], v);
          }
        }
      }
  if constexpr (Epi::kRowStats) {
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
        epi.row_stats(pe, r, blockIdx.x, red_sum[0][rl] + red_sum[1][rl],
                      fmaxf(red_max[0][rl], red_max[1][rl]));
    }
  }
}

// Large bf16 contractions: 128 x 128 tiles on 32x32x16 MFMA, each of the
// four waves a 64 x 64 quarter (2 x 2 MFMA tiles, every LDS fragment feeding
// two MFMAs), three register stages of 64-wide k slabs ahead, double-buffered
// LDS (dynamic, 72 KB).  Workgroups are dealt to the eight XCDs round robin,
// so workgroup b takes entry (b % 8) * per + b / 8 of the (problem, row tile,
// column tile) sequence and each XCD's L2 serves one contiguous range of it.
// Epilogues without row statistics only.
constexpr int kBigTile = 128;
constexpr int kBigStages = 3;
constexpr size_t kBigLds = 4ull * kBigTile * (kBK + 8) * sizeof(bf16_t);

template <class Epi>
__global__ void __launch_bounds__(256, 2)
gemm_nt_big_kernel(RowOperand<bf16_t> A, RowOperand<bf16_t> B, int K, int batch, Epi epi) {
  static_assert(!Epi::kRowStats, "row statistics need the 64-tile kernel");
  typedef float floatx16 __attribute__((ext_vector_type(16)));
  constexpr int BT = kBigTile, P = kBK + 8, CPR = kBK / 8, CH = BT * CPR / 256, S = kBigStages;
  extern __shared__ __attribute__((aligned(16))) unsigned char gemm_big_lds[];
  bf16_t* As = reinterpret_cast<bf16_t*>(gemm_big_lds);   // [2][BT * P]
  bf16_t* Bs = As + 2 * BT * P;                           // [2][BT * P]
  const int ntr = (A.rows + BT - 1) / BT, ntc = (B.rows + BT - 1) / BT, ntiles = ntr * ntc;
  const int per = (ntiles * batch + 7) / 8;
  const int f = (blockIdx.x % 8) * per + blockIdx.x / 8;
  if (f >= ntiles * batch) return;
  const int p = f / ntiles, t = f % ntiles;
  const int row0 = (t / ntc) * BT, col0 = (t % ntc) * BT;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;
  const bf16_t* a_src[CH];
  const bf16_t* b_src[CH];
#pragma unroll
  for (int q = 0; q < CH; ++q) {
    const int ch = tid + q * 256, r = ch / CPR, kc = (ch % CPR) * 8;
    a_src[q] = A.row(p, min(row0 + r, A.rows - 1)) + kc;
    b_src[q] = B.row(p, min(col0 + r, B.rows - 1)) + kc;
  }
  uint4 ra[S][CH], rb[S][CH];
  const int nk = K / kBK;
  auto load = [&](int kt, uint4* xa, uint4* xb) {
    const int k0 = min(kt, nk - 1) * kBK;
#pragma unroll
    for (int q = 0; q < CH; ++q) { xa[q] = ld16(a_src[q] + k0); xb[q] = ld16(b_src[q] + k0); }
  };
  auto store = [&](int buf, const uint4* xa, const uint4* xb) {
#pragma unroll
    for (int q = 0; q < CH; ++q) {
      const int ch = tid + q * 256, r = ch / CPR, kc = (ch % CPR) * 8;
      st16(&As[buf * BT * P + r * P + kc], xa[q]);
      st16(&Bs[buf * BT * P + r * P + kc], xb[q]);
    }
  };
  floatx16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
  // operand fragment of lane l: row l % 32 of a 32-row tile, k elements
  // 8 (l / 32) .. + 8 of the 16-wide step
  const int fr = lane & 31, fk = (lane >> 5) * 8;
  auto compute = [&](int buf) {
    const bf16_t* as = As + buf * BT * P;
    const bf16_t* bs = Bs + buf * BT * P;
#pragma unroll
    for (int ks = 0; ks < kBK; ks += 16) {
      bf16x8 fa[2], fb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        fa[i] = __builtin_bit_cast(bf16x8, ld16(&as[(wr * 64 + i * 32 + fr) * P + ks + fk]));
#pragma unroll
      for (int j = 0; j < 2; ++j)
        fb[j] = __builtin_bit_cast(bf16x8, ld16(&bs[(wc * 64 + j * 32 + fr) * P + ks + fk]));
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
  };
#pragma unroll
  for (int s = 0; s < S; ++s) load(s, ra[s], rb[s]);
  store(0, ra[0], rb[0]);
  __syncthreads();
  // whole groups of S steps (static register stages); S is odd, so the LDS
  // buffer follows the slab's own parity
  const int nk_main = nk - nk % S;
  for (int kt = 0; kt < nk_main; kt += S) {
#pragma unroll
    for (int s = 0; s < S; ++s) {
      load(kt + s + S, ra[s], rb[s]);
      compute((kt + s) & 1);
      store((kt + s + 1) & 1, ra[(s + 1) % S], rb[(s + 1) % S]);
      __syncthreads();
    }
  }
#pragma unroll
  for (int s = 0; s < S - 1; ++s) {
    if (nk_main + s >= nk) break;
    compute((nk_main + s) & 1);
    store((nk_main + s + 1) & 1, ra[(s + 1) % S], rb[(s + 1) % S]);
    __syncthreads();
  }
  // epilogue: acc[i][j][4 a + b] is C[32 i + 8 a + 4 (l / 32) + b][32 j + l % 32]
  // of the wave's quarter
  const int h = lane >> 5, cl = lane & 31;
  const int qr0 = row0 + wr * 64, qc0 = col0 + wc * 64;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int c = qc0 + 32 * j + cl;
    if (c >= B.rows) continue;
    const float csc = epi.col_scale(p, c);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int r = qr0 + 32 * i + 8 * a + 4 * h + b;
          if (r < A.rows) epi.value(p, r, c, acc[i][j][4 * a + b] * epi.row_scale(p, r) * csc);
        }
  }
}

template <class Epi>
inline hipError_t launch_gemm_nt_big(const RowOperand<bf16_t>& A, const RowOperand<bf16_t>& B, int K, int batch,
                                     const Epi& epi, hipStream_t stream) {
  if (K % kBK != 0) return hipErrorInvalidValue;
  static bool granted = false;
  if (!granted) {
    const hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(gemm_nt_big_kernel<Epi>),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(kBigLds));
    if (err != hipSuccess) return err;
    granted = true;
  }
  const long long tiles = static_cast<long long>((A.rows + kBigTile - 1) / kBigTile) *
                          ((B.rows + kBigTile - 1) / kBigTile) * batch;
  hipLaunchKernelGGL((gemm_nt_big_kernel<Epi>), dim3(static_cast<unsigned>((tiles + 7) / 8 * 8)), dim3(256), kBigLds,
                     stream, A, B, K, batch, epi);
  return hipGetLastError();
}

// K must divide into ksplit slices that are multiples of 64; with ksplit > 1
// the epilogue's problem index is problem * ksplit + split.
template <typename T, int BM, int BN, class Epi>
inline hipError_t launch_gemm_nt(const RowOperand<T>& A, const RowOperand<T>& B, int K, int batch,
                                 const Epi& epi, hipStream_t stream, int ksplit = 1) {
  if (ksplit < 1 || K % (kBK * ksplit) != 0) return hipErrorInvalidValue;
  dim3 grid((B.rows + BN - 1) / BN, (A.rows + BM - 1) / BM, batch * ksplit);
  hipLaunchKernelGGL((gemm_nt_kernel<T, BM, BN, Epi>), grid, dim3(kGemmThreads), 0, stream, A, B, K / ksplit,
                     ksplit, epi);
  return hipGetLastError();
}

}  // namespace gmc
