// Appearance and spatial client banks (Sec. 3.2; App. H Eq. cond-aux-clients,
// Eq. cond-coverage, Eq. cond-effective-bank-mass).
//
// Exact bank (N <= threshold): E_V[m][i] = exp((cos_mi - 1) / tau_v) from an
// MFMA Gram of the raw states (upper-triangle tiles only, mirrored in the
// epilogue), normalised after the contraction (cos = h_m.h_i / (|h_m| |h_i|))
// so the MFMA operands are the exact inputs.
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

// Exact bank on the symmetric Gram: only tiles (I, J) with I <= J of the
// 64 x 64 tiling are computed; each writes E_V for (client r in I, token c in
// J) and, off the diagonal, the mirror (client c, token r), with the row
// statistics of both orientations (client r over column block J; client c
// over column block I), so the N x N bank costs half the contraction.
// Same operand pipeline as the generic MFMA GEMM (two register stages, double
// LDS buffer), 256 threads in a 2 x 2 wave grid of 32 x 32 sub-tiles.
template <typename T>
__global__ void __launch_bounds__(kGemmThreads)
gram_sym_kernel(Shape sh, Ws ws, const T* hidden, float inv_tau, float norm_eps) {
  constexpr int BM = 64, EPC = 16 / sizeof(T), P = kBK + EPC, CPR = kBK / EPC;
  constexpr int CH = BM * CPR / kGemmThreads;   // chunks per thread per slab (A and B each)
  constexpr int WM = 32, TM = 2;
  __shared__ __attribute__((aligned(16))) T As[2][BM * P];
  __shared__ __attribute__((aligned(16))) T Bs[2][BM * P];
  __shared__ float rs_sum[2][BM], rs_max[2][BM], cs_sum[2][BM], cs_max[2][BM];
  // upper-triangle tile (I, J), I <= J, of problem p from the linear block
  // index, in XCD-contiguous order: workgroups go to the eight XCDs round
  // robin, so workgroup b takes entry (b % 8) * per + b / 8 of the (problem,
  // tile) sequence and each XCD works through one contiguous range, whose
  // tiles share operand rows in its own L2
  const int nt = (sh.N + BM - 1) / BM, ntiles = nt * (nt + 1) / 2;
  const int per = (ntiles * sh.B + 7) / 8;
  const int f = (blockIdx.x % 8) * per + blockIdx.x / 8;
  if (f >= ntiles * sh.B) return;
  const int p = f / ntiles;
  int I = 0, rem = f % ntiles;
  while (rem >= nt - I) { rem -= nt - I; ++I; }
  const int J = I + rem;
  const int row0 = I * BM, col0 = J * BM;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;
  const T* base = hidden + static_cast<long long>(p) * sh.N * sh.d;
  const T* a_src[CH];
  const T* b_src[CH];
#pragma unroll
  for (int q = 0; q < CH; ++q) {
    const int ch = tid + q * kGemmThreads, r = ch / CPR, kc = (ch % CPR) * EPC;
    a_src[q] = base + static_cast<long long>(min(row0 + r, sh.N - 1)) * sh.d + kc;
    b_src[q] = base + static_cast<long long>(min(col0 + r, sh.N - 1)) * sh.d + kc;
  }
  constexpr int S = gemm_stages<T>();
  uint4 ra[S][CH], rb[S][CH];
  const int nk = sh.d / kBK;
  auto load = [&](int kt, uint4* ra, uint4* rb) {
    const int k0 = min(kt, nk - 1) * kBK;
#pragma unroll
    for (int q = 0; q < CH; ++q) { ra[q] = ld16(a_src[q] + k0); rb[q] = ld16(b_src[q] + k0); }
  };
  auto store = [&](int buf, const uint4* ra, const uint4* rb) {
#pragma unroll
    for (int q = 0; q < CH; ++q) {
      const int ch = tid + q * kGemmThreads, r = ch / CPR, kc = (ch % CPR) * EPC;
      st16(&As[buf][r * P + kc], ra[q]);
      st16(&Bs[buf][r * P + kc], rb[q]);
    }
  };
  floatx4 acc[TM][TM];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int fr = lane & 15, fk = (lane >> 4) * 8;
  auto compute = [&](int buf) {
#pragma unroll
    for (int ks = 0; ks < kBK; ks += 32) {
      Frag<T> fa[TM], fb[TM];
#pragma unroll
      for (int i = 0; i < TM; ++i) fa[i] = frag_load<T>(&As[buf][(wr * WM + i * 16 + fr) * P + ks + fk]);
#pragma unroll
      for (int j = 0; j < TM; ++j) fb[j] = frag_load<T>(&Bs[buf][(wc * WM + j * 16 + fr) * P + ks + fk]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j) acc[i][j] = mma(fa[i], fb[j], acc[i][j]);
    }
  };
  // the GEMM core's slab pipeline: S register stages, double-buffered LDS
#pragma unroll
  for (int s = 0; s < S; ++s) load(s, ra[s], rb[s]);
  store(0, ra[0], rb[0]);
  __syncthreads();
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

  // epilogue: lane holds column (lane & 15), rows 4 (lane >> 4) + e of each
  // 16 x 16 tile; cos = acc / (|h_r| |h_c|), v = exp((cos - 1) / tau_v)
  const int oc = lane & 15, orow = (lane >> 4) * 4;
  const float* n2 = ws.n2 + p * ws.s_n;
  float rsc[TM][4], csc[TM];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e)
      rsc[i][e] = 1.f / fmaxf(sqrtf(n2[min(row0 + wr * WM + i * 16 + orow + e, sh.N - 1)]), norm_eps);
#pragma unroll
  for (int j = 0; j < TM; ++j) csc[j] = 1.f / fmaxf(sqrtf(n2[min(col0 + wc * WM + j * 16 + oc, sh.N - 1)]), norm_eps);
  // several images: a client covers its own image's tokens only
  int rim[TM][4], cim[TM];
  const int* img = ws.img + p * ws.s_img;
  const bool multi = sh.nimg > 1;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) rim[i][e] = multi ? img[min(row0 + wr * WM + i * 16 + orow + e, sh.N - 1)] : 0;
#pragma unroll
  for (int j = 0; j < TM; ++j) cim[j] = multi ? img[min(col0 + wc * WM + j * 16 + oc, sh.N - 1)] : 0;
  float* E = ws.E + p * ws.s_E;
  const bool diag = I == J;
  float rsum[TM][4], rmax[TM][4], csum[TM], cmax[TM];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) { rsum[i][e] = 0.f; rmax[i][e] = 0.f; }
#pragma unroll
  for (int j = 0; j < TM; ++j) { csum[j] = 0.f; cmax[j] = 0.f; }
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = row0 + wr * WM + i * 16 + orow + e;
        const int c = col0 + wc * WM + j * 16 + oc;
        if (r < sh.N && c < sh.N) {
          const float v = rim[i][e] == cim[j] ? expf((acc[i][j][e] * rsc[i][e] * csc[j] - 1.f) * inv_tau) : 0.f;
          E[static_cast<long long>(c) * sh.ldM + sh.mg + r] = v;           // client r, token c
          rsum[i][e] += v;
          rmax[i][e] = fmaxf(rmax[i][e], v);
          if (!diag) {
            E[static_cast<long long>(r) * sh.ldM + sh.mg + c] = v;         // client c, token r
            csum[j] += v;
            cmax[j] = fmaxf(cmax[j], v);
          }
        }
      }
  // client r: sum / max over the tile's columns (16 lanes of a row group,
  // then the two column waves); client c: over the tile's rows (4 rows per
  // lane, the 4 row groups, the two row tiles, then the two row waves)
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float sv = rsum[i][e], mv = rmax[i][e];
      sv = group16_sum(sv);
      mv = group16_max(mv);
      if (oc == 0) { rs_sum[wc][wr * WM + i * 16 + orow + e] = sv; rs_max[wc][wr * WM + i * 16 + orow + e] = mv; }
    }
  if (!diag) {
#pragma unroll
    for (int j = 0; j < TM; ++j) {
      float sv = csum[j], mv = cmax[j];
      sv = add_xor16(sv);
      mv = fmaxf(mv, xor_lane<16>(mv));
      sv = add_xor32(sv);
      mv = fmaxf(mv, xor_lane<32>(mv));
      if (lane < 16) { cs_sum[wr][wc * WM + j * 16 + oc] = sv; cs_max[wr][wc * WM + j * 16 + oc] = mv; }
    }
  }
  __syncthreads();
  float* ps = ws.apart_sum + p * ws.s_apart;
  float* pm = ws.apart_max + p * ws.s_apart;
  if (tid < BM) {
    const int r = row0 + tid;
    if (r < sh.N) {
      ps[static_cast<long long>(J) * sh.mv + r] = rs_sum[0][tid] + rs_sum[1][tid];
      pm[static_cast<long long>(J) * sh.mv + r] = fmaxf(rs_max[0][tid], rs_max[1][tid]);
    }
  } else if (!diag && tid < 2 * BM) {
    const int cl = tid - BM, c = col0 + cl;
    if (c < sh.N) {
      ps[static_cast<long long>(I) * sh.mv + c] = cs_sum[0][cl] + cs_sum[1][cl];
      pm[static_cast<long long>(I) * sh.mv + c] = fmaxf(cs_max[0][cl], cs_max[1][cl]);
    }
  }
}

// The exact bank for many tiles (bf16 states): 128 x 128 upper-triangle
// tiles of the Gram on 32x32x16 MFMA, each wave a 64 x 64 quarter (2 x 2
// MFMA tiles, so every LDS operand fragment feeds two MFMAs of 32K flop).
// Operands: 64-wide k slabs, three register stages ahead, double-buffered
// LDS.  The quarters are aligned with the 64-column blocks of the row
// statistics: quarter (a, b) of tile (I, J) is the 64 x 64 block pair
// (2I + a, 2J + b), written for (client r, token c) and, unless it is a
// diagonal block, mirrored; on a diagonal tile the lower quarter (1, 0)
// mirrors (0, 1) and writes nothing.  Row statistics per quarter go through
// LDS: one lane per client row (or column) of the quarter.
constexpr int kBigT = 128;
constexpr int kBigS = 3;
__global__ void __launch_bounds__(256, 2)
gram_sym_big_kernel(Shape sh, Ws ws, const bf16_t* hidden, float inv_tau, float norm_eps) {
  typedef float floatx16 __attribute__((ext_vector_type(16)));
  constexpr int BT = kBigT, P = kBK + 8, CPR = kBK / 8, CH = BT * CPR / 256, S = kBigS;
  extern __shared__ __attribute__((aligned(16))) unsigned char big_lds[];
  bf16_t* As = reinterpret_cast<bf16_t*>(big_lds);          // [2][BT * P]
  bf16_t* Bs = As + 2 * BT * P;                              // [2][BT * P]
  const int nt = (sh.N + BT - 1) / BT, ntiles = nt * (nt + 1) / 2;
  // XCD-contiguous order: workgroups go to the eight XCDs round robin, so
  // workgroup b takes entry (b % 8) * per + b / 8 of the (problem, tile)
  // sequence; each XCD then works through one contiguous range, whose tiles
  // share operand rows in its own L2
  const int per = (ntiles * sh.B + 7) / 8;
  const int f = (blockIdx.x % 8) * per + blockIdx.x / 8;
  if (f >= ntiles * sh.B) return;
  const int p = f / ntiles;
  int I = 0, rem = f % ntiles;
  while (rem >= nt - I) { rem -= nt - I; ++I; }
  const int J = I + rem;
  const int row0 = I * BT, col0 = J * BT;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;
  const bf16_t* base = hidden + static_cast<long long>(p) * sh.N * sh.d;
  const bf16_t* a_src[CH];
  const bf16_t* b_src[CH];
#pragma unroll
  for (int q = 0; q < CH; ++q) {
    const int ch = tid + q * 256, r = ch / CPR, kc = (ch % CPR) * 8;
    a_src[q] = base + static_cast<long long>(min(row0 + r, sh.N - 1)) * sh.d + kc;
    b_src[q] = base + static_cast<long long>(min(col0 + r, sh.N - 1)) * sh.d + kc;
  }
  uint4 ra[S][CH], rb[S][CH];
  const int nk = sh.d / kBK;
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
  // operand fragment of lane l: row l % 32 of the 32-row tile, k elements
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
  // whole groups of S steps (static register stages, no exit inside a group)
  const int nk_main = nk - nk % S;
  // (S is odd, so the LDS buffer follows the slab's own parity)
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

  // epilogue.  acc[i][j][4 a + b] is C[32 i + 8 a + 4 (l / 32) + b][32 j + l % 32]
  // of the quarter; v = exp((cos - 1) / tau_v), zero across images
  const bool diag_tile = I == J;
  const bool skip = diag_tile && wr == 1 && wc == 0;   // mirror of quarter (0, 1)
  const bool mirror = !(diag_tile && wr == wc);
  const int qr0 = row0 + wr * 64, qc0 = col0 + wc * 64;
  const float* n2 = ws.n2 + p * ws.s_n;
  const int* img = ws.img + p * ws.s_img;
  const bool multi = sh.nimg > 1;
  float* E = ws.E + p * ws.s_E;
  float* vt = reinterpret_cast<float*>(big_lds) + wave * 64 * 65;   // the quarter's values, pitch 65
  const int h = lane >> 5, cl = lane & 31;
  if (!skip) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int c = qc0 + 32 * j + cl;
      const bool cok = c < sh.N;
      const int cc = min(c, sh.N - 1);
      const float csc = 1.f / fmaxf(sqrtf(n2[cc]), norm_eps);
      const int cim = multi ? img[cc] : 0;
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          float v4[4];
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const int rl = 32 * i + 8 * a + 4 * h + b, r = qr0 + rl;
            const int rr = min(r, sh.N - 1);
            const float rsc = 1.f / fmaxf(sqrtf(n2[rr]), norm_eps);
            const bool ok = cok && r < sh.N && (!multi || img[rr] == cim);
            const float v = ok ? expf((acc[i][j][4 * a + b] * rsc * csc - 1.f) * inv_tau) : 0.f;
            v4[b] = v;
            vt[rl * 65 + 32 * j + cl] = v;
            if (mirror && cok && r < sh.N) E[static_cast<long long>(r) * sh.ldM + sh.mg + c] = v;   // client c, token r
          }
          const int r0 = qr0 + 32 * i + 8 * a + 4 * h;
          if (cok) {
            float* dst = E + static_cast<long long>(c) * sh.ldM + sh.mg + r0;   // client r, token c
            if (r0 + 3 < sh.N) {
              *reinterpret_cast<float4*>(dst) = make_float4(v4[0], v4[1], v4[2], v4[3]);
            } else {
#pragma unroll
              for (int b = 0; b < 4; ++b)
                if (r0 + b < sh.N) dst[b] = v4[b];
            }
          }
        }
    }
  }
  __syncthreads();   // every wave's quarter is in LDS (the operand buffers are done)
  if (!skip) {
    float* ps = ws.apart_sum + p * ws.s_apart;
    float* pm = ws.apart_max + p * ws.s_apart;
    // client r = qr0 + lane over the quarter's 64 columns (column block 2J + wc)
    if (qc0 < sh.N) {
      float sv = 0.f, mv = 0.f;
#pragma unroll 8
      for (int x = 0; x < 64; ++x) { const float v = vt[lane * 65 + x]; sv += v; mv = fmaxf(mv, v); }
      const int r = qr0 + lane;
      if (r < sh.N) {
        ps[static_cast<long long>(2 * J + wc) * sh.mv + r] = sv;
        pm[static_cast<long long>(2 * J + wc) * sh.mv + r] = mv;
      }
    }
    // client c = qc0 + lane over the quarter's 64 rows (row block 2I + wr)
    if (mirror && qr0 < sh.N) {
      float sv = 0.f, mv = 0.f;
#pragma unroll 8
      for (int x = 0; x < 64; ++x) { const float v = vt[x * 65 + lane]; sv += v; mv = fmaxf(mv, v); }
      const int c = qc0 + lane;
      if (c < sh.N) {
        ps[static_cast<long long>(2 * I + wr) * sh.mv + c] = sv;
        pm[static_cast<long long>(2 * I + wr) * sh.mv + c] = mv;
      }
    }
  }
}

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

// Normalise projected rows: one wave per token.  The same grid (N / 4
// blocks of 256 threads, N >= M_V) also lists the bounded bank's client
// tokens m_k = floor(k N / M_V).
__global__ void __launch_bounds__(256) normalize_rows_kernel(Shape sh, Params pr, Ws ws) {
  const int p = blockIdx.y, i = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int k = blockIdx.x * 256 + threadIdx.x;
  if (k < sh.mv) ws.clients[p * ws.s_cl + k] = static_cast<int>((static_cast<long long>(k) * sh.N) / sh.mv);
  if (i >= sh.N) return;
  float* y = ws.y + p * ws.s_y + static_cast<long long>(i) * sh.app_rank;
  float s = 0.f;
  for (int c = lane; c < sh.app_rank; c += 64) s += y[c] * y[c];
  s = wave_sum(s);
  const float inv = 1.f / fmaxf(sqrtf(s), pr.norm_eps);
  for (int c = lane; c < sh.app_rank; c += 64) y[c] *= inv;
}

// Appearance row weights alpha = (beta_app / M_V) / Z_m and peaks.
// 64 client rows per block (lane = row); wave w adds the column blocks
// [w nb/4, (w+1) nb/4) in order, then the four partial sums are added in
// wave order.
__global__ void __launch_bounds__(256) appearance_alpha_kernel(Shape sh, Params pr, Ws ws) {
  __shared__ float ps4[4][64], pm4[4][64];
  const int p = blockIdx.y, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = blockIdx.x * 64 + lane, rc = min(r, sh.mv - 1);
  const float* ps = ws.apart_sum + p * ws.s_apart;
  const float* pm = ws.apart_max + p * ws.s_apart;
  const int per = (sh.n_app_cblk + 3) / 4, b0 = wave * per, b1 = min(sh.n_app_cblk, b0 + per);
  float s = 0.f, m = 0.f;
#pragma unroll 8
  for (int b = b0; b < b1; ++b) {
    s += ps[static_cast<long long>(b) * sh.mv + rc];
    m = fmaxf(m, pm[static_cast<long long>(b) * sh.mv + rc]);
  }
  ps4[wave][lane] = s;
  pm4[wave][lane] = m;
  __syncthreads();
  if (wave == 0 && r < sh.mv) {
    s = ((ps4[0][lane] + ps4[1][lane]) + ps4[2][lane]) + ps4[3][lane];
    m = fmaxf(fmaxf(pm4[0][lane], pm4[1][lane]), fmaxf(pm4[2][lane], pm4[3][lane]));
    const float a = pr.beta_app / static_cast<float>(sh.mv) / s;
    ws.alpha[p * ws.s_m + sh.mg + r] = a;
    ws.peak[p * ws.s_m + sh.mg + r] = a * m;
  }
}

// Spatial bank, landmark side: one block per landmark l_ab = ((a+.5)/L,
// (b+.5)/L) of image g (row g L^2 + a L + b; one image: g = 0).  The block
// first takes the grid origin and extent of (h, w) over the image's tokens
// (temporal id excluded) and places each token at its cell centre in
// [0,1]^2; then the minimum squared distance to any token of the image, the
// row sum of exp(-(d^2 - min d^2)/tau_s), the weight (beta_spa / M_S) / Z and
// the peak (the row maximum is exactly 1).  The image's first landmark block
// also stores the token coordinates for the token-side kernel.
__device__ __forceinline__ float2 cell_centre(const int32_t* pos, int i, float h0, float w0, float gh, float gw) {
  return make_float2((static_cast<float>(pos[i * 3 + 1]) - h0 + 0.5f) / gh,
                     (static_cast<float>(pos[i * 3 + 2]) - w0 + 0.5f) / gw);
}

__global__ void __launch_bounds__(256) spatial_stats_kernel(Shape sh, Params pr, Ws ws, const int32_t* pos3d) {
  __shared__ float red[16];
  __shared__ float4 ext4[4];
  const int row = blockIdx.x, p = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = sh.landmarks, L2 = L * L;
  const int g = row / L2, lr = row % L2;
  const float ly = (static_cast<float>(lr / L) + 0.5f) / L;
  const float lx = (static_cast<float>(lr % L) + 0.5f) / L;
  const int32_t* pos = pos3d + static_cast<long long>(p) * sh.N * 3;
  const int* img = ws.img + p * ws.s_img;
  const bool multi = sh.nimg > 1;
  // the image's extents: one four-value block reduction
  float hmin = INFINITY, hmax = -INFINITY, wmin = INFINITY, wmax = -INFINITY;
  for (int i = tid; i < sh.N; i += blockDim.x) {
    if (multi && img[i] != g) continue;
    const float hh = static_cast<float>(pos[i * 3 + 1]), ww = static_cast<float>(pos[i * 3 + 2]);
    hmin = fminf(hmin, hh); hmax = fmaxf(hmax, hh);
    wmin = fminf(wmin, ww); wmax = fmaxf(wmax, ww);
  }
  hmin = wave_min(hmin); hmax = wave_max(hmax);
  wmin = wave_min(wmin); wmax = wave_max(wmax);
  if (lane == 0) ext4[wave] = make_float4(hmin, hmax, wmin, wmax);
  __syncthreads();
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float4 e = ext4[w];
    hmin = fminf(hmin, e.x); hmax = fmaxf(hmax, e.y);
    wmin = fminf(wmin, e.z); wmax = fmaxf(wmax, e.w);
  }
  const float gh = hmax - hmin + 1.f, gw = wmax - wmin + 1.f;
  // one pass for the minimum and the row sum: each thread keeps its own
  // running minimum m and the sum of exp(-(d^2 - m)/tau_s) relative to it
  // (rescaled when m drops); the sums are then brought to the block minimum
  const float inv_tau = 1.f / pr.tau_s;
  float* pc = ws.pc + p * ws.s_pc;
  float mt = INFINITY, st = 0.f;
  for (int i = tid; i < sh.N; i += blockDim.x) {
    if (multi && img[i] != g) continue;
    const float2 c = cell_centre(pos, i, hmin, wmin, gh, gw);
    const float dy = c.x - ly, dx = c.y - lx;
    const float d2 = dy * dy + dx * dx;
    if (d2 < mt) {
      st = (mt == INFINITY ? 0.f : st * expf(-(mt - d2) * inv_tau)) + 1.f;
      mt = d2;
    } else {
      st += expf(-(d2 - mt) * inv_tau);
    }
    if (lr == 0) {
      pc[2 * i] = c.x;
      pc[2 * i + 1] = c.y;
    }
  }
  const float dmin = block_min(mt, red);
  const float s = block_sum(mt == INFINITY ? 0.f : st * expf(-(mt - dmin) * inv_tau), red);
  if (tid == 0) {
    const int m = sh.mg + sh.mv + row;
    // an image without tokens (reported by the input status bit) keeps an
    // inert row
    const float a = s > 0.f ? pr.beta_spa / static_cast<float>(sh.ms) / s : 0.f;
    ws.alpha[p * ws.s_m + m] = a;
    ws.peak[p * ws.s_m + m] = a;
    ws.lstat[p * ws.s_lstat + row] = s > 0.f ? dmin : 0.f;
  }
}

// Spatial bank, token side: one wave per token writes its landmark energies,
// contiguous in the token-major client matrix (zero for the landmarks of
// other images).
__global__ void __launch_bounds__(256) spatial_write_kernel(Shape sh, Params pr, Ws ws) {
  const int p = blockIdx.y, i = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (i >= sh.N) return;
  const int L = sh.landmarks, L2 = L * L;
  const float* pc = ws.pc + p * ws.s_pc;
  const float py = pc[2 * i], px = pc[2 * i + 1];
  const int gi = sh.nimg > 1 ? ws.img[p * ws.s_img + i] : 0;
  const float inv_tau = 1.f / pr.tau_s;
  const float* dmin = ws.lstat + p * ws.s_lstat;
  float* E = ws.E + p * ws.s_E + static_cast<long long>(i) * sh.ldM + sh.mg + sh.mv;
  for (int row = lane; row < sh.ms; row += 64) {
    const int lr = row % L2;
    const float ly = (static_cast<float>(lr / L) + 0.5f) / L;
    const float lx = (static_cast<float>(lr % L) + 0.5f) / L;
    const float dy = py - ly, dx = px - lx;
    E[row] = (row / L2 == gi) ? expf(-(dy * dy + dx * dx - dmin[row]) * inv_tau) : 0.f;
  }
}

// Spatial bank in one launch (up to kSpatialFusedN tokens per call, all
// problems together): one block per landmark row with the landmark-side
// kernel's statistics (the minimum and the row sum in two passes here), and
// the block then writes its row's energies itself: one 4-byte value per
// token row of the client matrix (zero for the tokens of other images).  Beyond kSpatialFusedN tokens those scattered stores cost
// more than the token-side kernel's contiguous rows and the second launch
// it needs (measured: one 1296-token image 14.5 against 16.0 us, sixteen
// of them 65 against 46 us).
constexpr int kSpatialFusedN = 2048;

__device__ __forceinline__ float sq_dist(float2 c, float ly, float lx) {
  const float dy = c.x - ly, dx = c.y - lx;
  return dy * dy + dx * dx;
}

__global__ void __launch_bounds__(256) spatial_bank_kernel(Shape sh, Params pr, Ws ws, const int32_t* pos3d) {
  __shared__ float red[16];
  __shared__ float4 ext4[4];
  const int row = blockIdx.x, p = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = sh.landmarks, L2 = L * L;
  const int g = row / L2, lr = row % L2;
  const float ly = (static_cast<float>(lr / L) + 0.5f) / L;
  const float lx = (static_cast<float>(lr % L) + 0.5f) / L;
  const int32_t* pos = pos3d + static_cast<long long>(p) * sh.N * 3;
  const int* img = ws.img + p * ws.s_img;
  const bool multi = sh.nimg > 1;
  float hmin = INFINITY, hmax = -INFINITY, wmin = INFINITY, wmax = -INFINITY;
  for (int i = tid; i < sh.N; i += 256) {
    if (multi && img[i] != g) continue;
    const float hh = static_cast<float>(pos[i * 3 + 1]), ww = static_cast<float>(pos[i * 3 + 2]);
    hmin = fminf(hmin, hh); hmax = fmaxf(hmax, hh);
    wmin = fminf(wmin, ww); wmax = fmaxf(wmax, ww);
  }
  hmin = wave_min(hmin); hmax = wave_max(hmax);
  wmin = wave_min(wmin); wmax = wave_max(wmax);
  if (lane == 0) ext4[wave] = make_float4(hmin, hmax, wmin, wmax);
  __syncthreads();
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float4 e = ext4[w];
    hmin = fminf(hmin, e.x); hmax = fmaxf(hmax, e.y);
    wmin = fminf(wmin, e.z); wmax = fmaxf(wmax, e.w);
  }
  const float gh = hmax - hmin + 1.f, gw = wmax - wmin + 1.f;
  float* pc = ws.pc + p * ws.s_pc;
  float dmin = INFINITY;
  for (int i = tid; i < sh.N; i += 256) {
    if (multi && img[i] != g) continue;
    const float2 c = cell_centre(pos, i, hmin, wmin, gh, gw);
    dmin = fminf(dmin, sq_dist(c, ly, lx));
    if (lr == 0) {
      pc[2 * i] = c.x;
      pc[2 * i + 1] = c.y;
    }
  }
  dmin = block_min(dmin, red);
  const float inv_tau = 1.f / pr.tau_s;
  float s = 0.f;
  for (int i = tid; i < sh.N; i += 256) {
    if (multi && img[i] != g) continue;
    s += expf(-(sq_dist(cell_centre(pos, i, hmin, wmin, gh, gw), ly, lx) - dmin) * inv_tau);
  }
  s = block_sum(s, red);
  if (tid == 0) {
    const int m = sh.mg + sh.mv + row;
    // an image without tokens (reported by the input status bit) keeps an
    // inert row
    const float a = s > 0.f ? pr.beta_spa / static_cast<float>(sh.ms) / s : 0.f;
    ws.alpha[p * ws.s_m + m] = a;
    ws.peak[p * ws.s_m + m] = a;
  }
  float* E = ws.E + p * ws.s_E + sh.mg + sh.mv + row;
  for (int i = tid; i < sh.N; i += 256) {
    const bool own = !multi || img[i] == g;
    const float d2 = own ? sq_dist(cell_centre(pos, i, hmin, wmin, gh, gw), ly, lx) : 0.f;
    E[static_cast<long long>(i) * sh.ldM] = own ? expf(-(d2 - dmin) * inv_tau) : 0.f;
  }
}

template <typename T>
static hipError_t banks_impl(const Shape& sh, const Params& pr, const Ws& ws, const void* hidden_v,
                             const void* proj_v, const int32_t* pos3d, hipStream_t st) {
  const T* hidden = static_cast<const T*>(hidden_v);
  hipError_t err;
  auto spatial = [&]() {
    timer_mark(kStSpatial, true, st);
    if (static_cast<long long>(sh.N) * sh.B <= kSpatialFusedN) {
      hipLaunchKernelGGL(spatial_bank_kernel, dim3(sh.ms, sh.B), dim3(256), 0, st, sh, pr, ws, pos3d);
    } else {
      hipLaunchKernelGGL(spatial_stats_kernel, dim3(sh.ms, sh.B), dim3(256), 0, st, sh, pr, ws, pos3d);
      hipLaunchKernelGGL(spatial_write_kernel, dim3((sh.N + 3) / 4, sh.B), dim3(256), 0, st, sh, pr, ws);
    }
    timer_mark(kStSpatial, false, st);
  };
  // up to 2048 tokens the light spatial kernels go first, so that the Gram,
  // the heaviest bank kernel, overlaps the head-pattern kernels rather than
  // the probe and the message logits (measured at 1296 tokens: the call
  // takes 289 us this way, 299 us with the Gram first, and the Gram's row
  // weights are ready within 1 us of the head clustering); a larger Gram
  // starts at once
  const bool spatial_first = sh.N <= 2048;
  if (spatial_first) spatial();
  timer_mark(kStAppearance, true, st);
  if (!sh.bounded) {
    const int nt = (sh.N + 63) / 64, nt2 = (sh.N + kBigT - 1) / kBigT;
    // 128-row tiles once they alone fill the chip twice over (bf16 states)
    bool big = false;
    if constexpr (sizeof(T) == 2) {
      if (static_cast<long long>(nt2) * (nt2 + 1) / 2 * sh.B >= 512) {
        constexpr size_t lds = 4ull * kBigT * (kBK + 8) * sizeof(bf16_t);
        static bool granted = false;
        if (!granted) {
          err = hipFuncSetAttribute(reinterpret_cast<const void*>(gram_sym_big_kernel),
                                    hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
          if (err != hipSuccess) return err;
          granted = true;
        }
        const int per = (nt2 * (nt2 + 1) / 2 * sh.B + 7) / 8;
        hipLaunchKernelGGL(gram_sym_big_kernel, dim3(8 * per), dim3(256), lds, st, sh, ws, hidden, 1.f / pr.tau_v,
                           pr.norm_eps);
        big = true;
      }
    }
    if (!big) {
      const int per = (nt * (nt + 1) / 2 * sh.B + 7) / 8;
      hipLaunchKernelGGL(gram_sym_kernel<T>, dim3(8 * per), dim3(kGemmThreads), 0, st, sh, ws, hidden,
                         1.f / pr.tau_v, pr.norm_eps);
    }
  } else {
    RowOperand<T> A{hidden, sh.d, static_cast<long long>(sh.N) * sh.d, nullptr, 0, sh.N};
    RowOperand<T> R{static_cast<const T*>(proj_v), sh.d, 0, nullptr, 0, sh.app_rank};
    ProjEpi pe{ws, sh.app_rank};
    err = launch_gemm_nt<T, 64, 64>(A, R, sh.d, sh.B, pe, st);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(normalize_rows_kernel, dim3((sh.N + 3) / 4, sh.B), dim3(256), 0, st, sh, pr, ws);
    RowOperand<float> Yc{ws.y, sh.app_rank, ws.s_y, ws.clients, ws.s_cl, sh.mv};
    RowOperand<float> Y{ws.y, sh.app_rank, ws.s_y, nullptr, 0, sh.N};
    AppearanceEpi epi{ws, sh.ldM, sh.mg, 0, 1.f / pr.tau_v, pr.norm_eps, sh.n_app_cblk, sh.mv};
    // small tiles: short blocks (a rank-long contraction each, four per CU
    // by LDS) interleave better with the message kernels running beside
    // them (measured on four 64 x 64 frames: the call 1% faster, the
    // kernel alone unchanged)
    err = launch_gemm_nt<float, kAppBoundedTile, kAppBoundedTile>(Yc, Y, sh.app_rank, sh.B, epi, st);
    if (err != hipSuccess) return err;
  }
  hipLaunchKernelGGL(appearance_alpha_kernel, dim3((sh.mv + 63) / 64, sh.B), dim3(256), 0, st, sh, pr, ws);
  timer_mark(kStAppearance, false, st);
  if (!spatial_first) spatial();
  return hipGetLastError();
}

hipError_t launch_banks(const Shape& sh, const Params& pr, const Ws& ws, const void* hidden,
                        const void* app_proj, const int32_t* pos3d, hipStream_t st) {
  if (sh.dtype == 0) return banks_impl<float>(sh, pr, ws, hidden, app_proj, pos3d, st);
  return banks_impl<bf16_t>(sh, pr, ws, hidden, app_proj, pos3d, st);
}

}  // namespace gmc
