// Batched responsibility selection (Sec. 3.3 Eq. coverage, Eq.
// responsibility; App. H Eq. cond-responsibility and the totality rule).
//
// The client energies are stored token-major, Et[i][m] (row stride ldM), and
// Cbar_mi = alpha_m Et[i][m] is formed on the fly.  Token-major makes every
// token's singleton gain u_i = sum_m [Cbar_mi - b_m]_+ one contiguous
// reduction owned by a single wave, so no cross-block partial sums exist.
// One round:
//   cov   - b_m <- max(b_m, max_{j in previous batch} Cbar_mj), rows in parallel,
//           batch columns split over blocks; in-place atomicMax on the bit
//           pattern (non-negative floats order like their bits), so the
//           result is independent of arrival order
//   gains - u_i per token; the last block picks the pool, the min(4b, N-|S|)
//           largest gains of unselected tokens (ties to the lower index)
//   resp  - pool of at most 64: one lane per client row computes the
//           responsibility softmax of R over the pool and its contributions
//           rho R; a butterfly transpose-reduction sums them per pool token;
//           the last block adds the block sums in order and picks the batch.
//           Larger pools (bounded path): per-row max and softmax denominator
//           first (rowstat), then one wave per pool token sums its column
//           (colsum), the last block picks the batch.
// Every reduction has a fixed order, so results are bitwise repeatable.
// Zero-gain tokens key just above excluded ones, so once gains vanish the
// lowest source indices fill the budget.
#include "gmc_device.h"
#include "gmc_internal.h"
#include "gmc_kernels.h"

namespace gmc {

constexpr int kCpw = 4;                 // gains kernel: tokens per wave
constexpr int kGainCols = 4 * kCpw;     // tokens per block
constexpr int kCpwF = 4;                // fused gains kernel: tokens per wave
constexpr int kGainColsF = 4 * kCpwF;
constexpr int kLdsKeys = 12288;         // pool top-k keys live in LDS up to this N

// Deterministic top-k over n keys (256-thread block): the `count` largest
// keys, equal keys resolved to the lower index.  Indices are written in
// ascending order to out[0..count).  count must not exceed the number of
// non-zero keys.  Radix selection of the threshold key with 8-bit digits
// (digits shared by every key are skipped; two histogram buffers, so each
// pass needs two block barriers), then one packed scan for the ordered
// compaction (each thread owns a contiguous index segment).
// hist: 512 ints of LDS, scan: >= 16 ints, bc: 2 ints.
__device__ void block_topk256(const uint32_t* keys, int n, int count, int* out, int* hist, int* scan,
                              int* bc) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  hist[tid] = 0;
  hist[256 + tid] = 0;
  uint32_t kand = 0xFFFFFFFFu, kor = 0u;
  for (int i = tid; i < n; i += 256) {
    const uint32_t k = keys[i];
    kand &= k;
    kor |= k;
  }
  kand = wave_and_u(kand);
  kor = wave_or_u(kor);
  if (lane == 0) { scan[wave] = static_cast<int>(kand); scan[4 + wave] = static_cast<int>(kor); }
  __syncthreads();
  kand = static_cast<uint32_t>(scan[0]) & static_cast<uint32_t>(scan[1]) & static_cast<uint32_t>(scan[2]) &
         static_cast<uint32_t>(scan[3]);
  kor = static_cast<uint32_t>(scan[4]) | static_cast<uint32_t>(scan[5]) | static_cast<uint32_t>(scan[6]) |
        static_cast<uint32_t>(scan[7]);
  const uint32_t diff = kand ^ kor;                 // bits that vary between keys
  uint32_t mask = 0;
  int top = 24;
  while (top > 0 && ((diff >> top) & 0xFFu) == 0u) {
    mask |= 0xFFu << top;
    top -= 8;
  }
  uint32_t prefix = kand & mask;
  int remaining = count, buf = 0;
  for (int shift = top; shift >= 0; shift -= 8, buf ^= 1) {
    int* h = hist + buf * 256;
    for (int i = tid; i < n; i += 256) {
      const uint32_t k = keys[i];
      if ((k & mask) == prefix) atomicAdd(&h[(k >> shift) & 255u], 1);
    }
    hist[(buf ^ 1) * 256 + tid] = 0;   // read in the previous pass; used by the next one
    __syncthreads();
    if (wave == 0) {
      // wave 0 scans the 256 bins from the top digit down, 4 per lane
      int v[4], loc = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) { v[q] = h[255 - (lane * 4 + q)]; loc += v[q]; }
      int excl = wave_scan_add(loc) - loc;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (excl < remaining && remaining <= excl + v[q]) {
          bc[0] = 255 - (lane * 4 + q);
          bc[1] = remaining - excl;
        }
        excl += v[q];
      }
    }
    __syncthreads();
    prefix |= static_cast<uint32_t>(bc[0]) << shift;
    mask |= 0xFFu << shift;
    remaining = bc[1];
  }
  const uint32_t kth = prefix;
  const int seg = (n + 255) / 256;
  const int i0 = min(n, tid * seg), i1 = min(n, i0 + seg);
  int gt = 0, eq = 0;
  for (int i = i0; i < i1; ++i) {
    const uint32_t k = keys[i];
    gt += k > kth;
    eq += k == kth;
  }
  int tot;
  const int pre = block_exclusive_scan(gt | (eq << 16), scan, &tot);
  int gt_b = static_cast<int>(static_cast<unsigned>(pre) & 0xFFFFu);
  int eq_b = static_cast<int>(static_cast<unsigned>(pre) >> 16);
  for (int i = i0; i < i1; ++i) {
    const uint32_t k = keys[i];
    if (k > kth) {
      out[gt_b + min(eq_b, remaining)] = i;
      ++gt_b;
    } else if (k == kth) {
      if (eq_b < remaining) out[gt_b + eq_b] = i;
      ++eq_b;
    }
  }
  __syncthreads();
}

// Register-resident variant of the same selection for small n: thread t
// holds the keys of its contiguous index segment [t*seg, t*seg + seg) in
// k[0..KPT) (0 past the segment; zero keys are excluded).  The radix windows
// start at the highest bit in which the non-zero keys differ, so the first
// histogram spreads the keys over up to 256 bins.  Passes continue until the
// bin holding the threshold is taken whole (the selection is then every
// non-zero key >= the resolved prefix) or every bit is resolved (the
// threshold is one key value, its first `remaining` copies by index taken).
// Every wave scans the histograms itself, so a radix pass needs one block
// barrier (three histogram buffers rotate).  The block has NW >= 4 waves.
// The selected indices are written to out[0, count) in ascending index order
// and out[count, fill) is filled with index 0.
// hist: 768 ints of LDS, scan: >= 3 NW ints.
template <int KPT, int NW = 4>
__device__ void block_topk_regs(const uint32_t (&k)[KPT], int seg, int count, int* out, int* hist, int* scan,
                                int fill = 64) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid < 256) {
    hist[tid] = 0;
    hist[256 + tid] = 0;
    hist[512 + tid] = 0;
  }
  uint32_t kand = 0xFFFFFFFFu, kor = 0u;
#pragma unroll
  for (int q = 0; q < KPT; ++q) {
    kand &= k[q] ? k[q] : 0xFFFFFFFFu;
    kor |= k[q];
  }
  kand = wave_and_u(kand);
  kor = wave_or_u(kor);
  if (lane == 0) { scan[wave] = static_cast<int>(kand); scan[NW + wave] = static_cast<int>(kor); }
  __syncthreads();
  kand = static_cast<uint32_t>(scan[0]);
  kor = static_cast<uint32_t>(scan[NW]);
#pragma unroll
  for (int w = 1; w < NW; ++w) {
    kand &= static_cast<uint32_t>(scan[w]);
    kor |= static_cast<uint32_t>(scan[NW + w]);
  }
  const uint32_t diff = kand ^ kor;
  // bits [hi, 32) are shared by every non-zero key; with no differing bit
  // every non-zero key equals kand
  int hi = diff ? 32 - __clz(diff) : 0;
  uint32_t mask = hi >= 32 ? 0u : ~((1u << hi) - 1u);
  uint32_t prefix = kand & mask;
  int remaining = count, buf = 0;
  while (hi > 0) {
    const int lo = max(hi - 8, 0);
    const uint32_t wmask = ((1u << (hi - lo)) - 1u) << lo;
    int* h = hist + buf * 256;
#pragma unroll
    for (int q = 0; q < KPT; ++q)
      if (k[q] != 0u && (k[q] & mask) == prefix) atomicAdd(&h[(k[q] & wmask) >> lo], 1);
    const int nxt = buf == 2 ? 0 : buf + 1;
    if (tid < 256) hist[nxt * 256 + tid] = 0;   // last read two passes ago
    __syncthreads();
    int v[4], loc = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) { v[q] = h[255 - (lane * 4 + q)]; loc += v[q]; }
    const int incl = wave_scan_add(loc);
    int excl = incl - loc;
    const bool hit = excl < remaining && remaining <= incl;
    int dig = 0, rem = 0, inbin = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (excl < remaining && remaining <= excl + v[q]) {
        dig = 255 - (lane * 4 + q);
        rem = remaining - excl;
        inbin = v[q];
      }
      excl += v[q];
    }
    const int src = __ffsll(static_cast<unsigned long long>(__ballot(hit))) - 1;
    dig = __builtin_amdgcn_readlane(dig, src);
    rem = __builtin_amdgcn_readlane(rem, src);
    inbin = __builtin_amdgcn_readlane(inbin, src);
    prefix |= static_cast<uint32_t>(dig) << lo;
    mask |= wmask;
    remaining = rem;
    hi = lo;
    if (inbin == remaining) {
      // every key of the threshold bin is taken: the selection is exactly
      // the non-zero keys >= prefix (its unresolved bits zero)
      remaining = count;
      hi = 0;
    }
    buf = nxt;
  }
  const uint32_t kth = prefix;
  int gt = 0, eq = 0;
#pragma unroll
  for (int q = 0; q < KPT; ++q) {
    gt += k[q] != 0u && k[q] > kth;
    eq += k[q] != 0u && k[q] == kth;
  }
  // exclusive prefix of (gt, eq) over threads: wave scans, then the wave
  // totals (scan[2 NW, 3 NW), untouched earlier in the call) after one barrier
  const int v = gt | (eq << 16);
  const int incl = wave_scan_add(v);
  if (lane == 63) scan[2 * NW + wave] = incl;
  __syncthreads();
  int pre = incl - v;
  for (int w = 0; w < wave; ++w) pre += scan[2 * NW + w];
  int gt_b = static_cast<int>(static_cast<unsigned>(pre) & 0xFFFFu);
  int eq_b = static_cast<int>(static_cast<unsigned>(pre) >> 16);
  const int i0 = tid * seg;
#pragma unroll
  for (int q = 0; q < KPT; ++q) {
    if (k[q] == 0u) continue;
    if (k[q] > kth) {
      out[gt_b + min(eq_b, remaining)] = i0 + q;
      ++gt_b;
    } else if (k[q] == kth) {
      if (eq_b < remaining) out[gt_b + eq_b] = i0 + q;
      ++eq_b;
    }
  }
  if (tid >= count && tid < fill) out[tid] = 0;
  __syncthreads();
}

// ---------------------------------------------------------------------------
// coverage refresh with a batch
// ---------------------------------------------------------------------------
constexpr int kCovCols = 32;   // batch columns per block

__global__ void __launch_bounds__(256) cov_kernel(Shape sh, Ws ws, int nb) {
  const int p = blockIdx.z, m = blockIdx.x * 256 + threadIdx.x;
  if (m >= sh.m) return;
  const int j0 = blockIdx.y * kCovCols, j1 = min(nb, j0 + kCovCols);
  const float a = ws.alpha[p * ws.s_m + m];
  const int* bat = ws.batch + p * ws.s_bat;
  const float* E = ws.E + p * ws.s_E + m;
  float c = 0.f;
  for (int j = j0; j < j1; ++j) c = fmaxf(c, a * E[static_cast<long long>(bat[j]) * sh.ldM]);
  atomicMax(reinterpret_cast<unsigned*>(&ws.cov[p * ws.s_cov + m]), __float_as_uint(c));
}

// ---------------------------------------------------------------------------
// singleton gains and the pool
// ---------------------------------------------------------------------------
// Singleton gains u_i = sum_m alpha_m max(E_mi - b_m, 0) of every token, four
// per wave; the client rows are streamed with non-temporal loads (the matrix
// is read once per round and is larger than the caches).  With kTail the last block to finish picks the pool itself (keys
// in LDS, or in global memory for large N); without it pool_topk_kernel
// follows.
template <bool kGlobalKeys, bool kTail = true>
__global__ void __launch_bounds__(256)
gains_kernel(Shape sh, Ws ws, int round, int psize, SelOut so) {
  extern __shared__ uint32_t keys_lds[];
  __shared__ int hist[512], scan[16], bc[2], flag;
  const int p = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int col0 = blockIdx.x * kGainCols + wave * kCpw;
  const float* alpha = ws.alpha + p * ws.s_m;
  const float* cov = ws.cov + p * ws.s_cov;
  const float* E = ws.E + p * ws.s_E;
  float* u = ws.u + p * ws.s_u;
  float acc[kCpw];
  const float* col[kCpw];
#pragma unroll
  for (int c = 0; c < kCpw; ++c) {
    acc[c] = 0.f;
    col[c] = E + static_cast<long long>(min(col0 + c, sh.N - 1)) * sh.ldM;
  }
#pragma unroll 4
  for (int m = lane * 4; m < sh.m; m += 256) {
    const float4 a = *reinterpret_cast<const float4*>(alpha + m);
    const float4 b = *reinterpret_cast<const float4*>(cov + m);
#pragma unroll
    for (int c = 0; c < kCpw; ++c) {
      const float4 v = ld_stream4(col[c] + m);
      acc[c] += fmaxf(a.x * v.x - b.x, 0.f);
      acc[c] += fmaxf(a.y * v.y - b.y, 0.f);
      acc[c] += fmaxf(a.z * v.z - b.z, 0.f);
      acc[c] += fmaxf(a.w * v.w - b.w, 0.f);
    }
  }
#pragma unroll
  for (int c = 0; c < kCpw; ++c) {
    const float s = wave_sum(acc[c]);
    if (lane == 0 && col0 + c < sh.N) st_dev(&u[col0 + c], s);
  }
  if constexpr (!kTail) return;

  // tail: the pool, the psize largest gains among unselected tokens
  int* cnt = ws.cnt + p * ws.s_cnt;
  if (!last_arrival(&cnt[0], gridDim.x, &flag)) return;
  if (tid == 0) st_dev(&cnt[0], 0);
  uint32_t* keys = kGlobalKeys ? ws.keys + p * ws.s_keys : keys_lds;
  const int* sel = ws.sel + p * ws.s_sel;
  // loads go to registers in batches first (keys may alias global memory, so
  // interleaved stores would serialise them)
  for (int base = 0; base < sh.N; base += 256 * 16) {
    float g[16];
    int sl[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int i = min(base + q * 256 + tid, sh.N - 1);
      g[q] = ld_dev(&u[i]);
      sl[q] = sel[i];
    }
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int i = base + q * 256 + tid;
      if (i < sh.N) {
        keys[i] = (sl[q] >= 0) ? 0u : score_key(g[q]);
        if (so.gains) so.gains[(static_cast<long long>(p) * sh.rounds + round) * sh.N + i] = (sl[q] >= 0) ? 0.f : g[q];
      }
    }
  }
  __syncthreads();
  int* pool = ws.pool + p * ws.s_pool;
  block_topk256(keys, sh.N, psize, pool, hist, scan, bc);
  if (so.pool) {
    int32_t* tp = so.pool + (static_cast<long long>(p) * sh.rounds + round) * sh.pool_cap;
    for (int j = tid; j < sh.pool_cap; j += 256) tp[j] = (j < psize) ? pool[j] : -1;
  }
}

// The pool of a per-round call: the psize largest gains among unselected
// tokens, ascending by index, equal gains resolved to the lower index (the
// same selection as the gains kernel's tail).  One 1024-thread block per
// problem: the keys are made from coalesced loads into LDS (dynamic, N
// words), then thread t takes tokens [t seg, t seg + seg) into registers
// (seg <= KPT), so every radix pass works on registers and LDS histograms.
constexpr int kPoolW = 16;   // waves of the pool top-k block
template <int KPT>
__global__ void __launch_bounds__(64 * kPoolW) pool_topk_kernel(Shape sh, Ws ws, int round, int psize,
                                                                 SelOut so) {
  extern __shared__ uint32_t keys_lds[];
  __shared__ int hist[768], scan[3 * kPoolW];
  const int p = blockIdx.x, tid = threadIdx.x;
  const float* u = ws.u + p * ws.s_u;
  const int* sel = ws.sel + p * ws.s_sel;
  constexpr int kT = 64 * kPoolW;
  float g[KPT];
  int sl[KPT];
#pragma unroll
  for (int q = 0; q < KPT; ++q) {
    const int i = min(q * kT + tid, sh.N - 1);
    g[q] = u[i];
    sl[q] = sel[i];
  }
#pragma unroll
  for (int q = 0; q < KPT; ++q) {
    const int i = q * kT + tid;
    if (i < sh.N) {
      keys_lds[i] = sl[q] < 0 ? score_key(g[q]) : 0u;
      if (so.gains) so.gains[(static_cast<long long>(p) * sh.rounds + round) * sh.N + i] = (sl[q] >= 0) ? 0.f : g[q];
    }
  }
  __syncthreads();
  const int seg = (sh.N + kT - 1) / kT;
  const int i0 = tid * seg;
  uint32_t k[KPT];
#pragma unroll
  for (int q = 0; q < KPT; ++q) k[q] = (q < seg && i0 + q < sh.N) ? keys_lds[i0 + q] : 0u;
  int* pool = ws.pool + p * ws.s_pool;
  block_topk_regs<KPT, kPoolW>(k, seg, psize, pool, hist, scan, 0);
  if (so.pool) {
    int32_t* tp = so.pool + (static_cast<long long>(p) * sh.rounds + round) * sh.pool_cap;
    for (int j = tid; j < sh.pool_cap; j += 64 * kPoolW) tp[j] = (j < psize) ? pool[j] : -1;
  }
}

// Mark the batch (indices into the pool, ascending) and record it.
__device__ void commit_batch(const Shape& sh, const Ws& ws, int p, int round, int bsize, int sel_base,
                             const int* pool_s, const int* chosen, int32_t* trace_batch) {
  int* sel = ws.sel + p * ws.s_sel;
  int* order = ws.order + p * ws.s_ord;
  int* batch = ws.batch + p * ws.s_bat;
  for (int k = threadIdx.x; k < bsize; k += blockDim.x) {
    const int i = pool_s[chosen[k]];
    sel[i] = round;
    order[sel_base + k] = i;
    batch[k] = i;
  }
  if (trace_batch) {
    int32_t* tb = trace_batch + (static_cast<long long>(p) * sh.rounds + round) * sh.b;
    for (int k = threadIdx.x; k < sh.b; k += blockDim.x) tb[k] = (k < bsize) ? pool_s[chosen[k]] : -1;
  }
}

// Ballot-based selection inside one wave.  Keys are held in lanes (KPT per
// lane); the count of keys >= c is a sum of ballot popcounts, so the
// count-th largest key value is found by a 32-step bitwise search with no
// LDS traffic: the largest v with at least `count` keys >= v.
template <int KPT>
__device__ __forceinline__ int wave_count_ge(const uint32_t (&k)[KPT], uint32_t c) {
  int n = 0;
#pragma unroll
  for (int q = 0; q < KPT; ++q) n += __popcll(__ballot(k[q] >= c));
  return n;
}
template <int KPT>
__device__ __forceinline__ uint32_t wave_kth(const uint32_t (&k)[KPT], int count) {
  uint32_t prefix = 0;
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t cand = prefix | (1u << bit);
    if (wave_count_ge<KPT>(k, cand) >= count) prefix = cand;
  }
  return prefix;
}

// Wave-level top-b of at most 64 keys (lane = pool position, ascending
// source index): rank by (key desc, position asc); chosen positions in
// ascending order.  Called by one whole wave.
__device__ void wave_topb(const uint32_t* keys, int psize, int bsize, int* chosen) {
  const int lane = threadIdx.x & 63;
  const unsigned long long below = (1ull << lane) - 1ull;
  const uint32_t k[1] = {(lane < psize) ? keys[lane] : 0u};
  const uint32_t kth = wave_kth<1>(k, bsize);
  const int quota = bsize - __popcll(__ballot(k[0] > kth));
  const unsigned long long eqm = __ballot(lane < psize && k[0] == kth);
  const bool take = lane < psize && (k[0] > kth || (k[0] == kth && __popcll(eqm & below) < quota));
  const unsigned long long tm = __ballot(take);
  if (take) chosen[__popcll(tm & below)] = lane;
}

// Butterfly transpose-reduction: lane l holds v[0..63] (one value per pool
// position); afterwards v[0] in lane l is the sum over all 64 lanes of the
// values for position l.  63 exchanges, fixed order.
template <int O>
__device__ __forceinline__ void transpose_reduce_step(float* v, int lane) {
  const bool hi = (lane & O) != 0;
#pragma unroll
  for (int k = 0; k < O; ++k) {
    const float send = hi ? v[k] : v[k + O];
    const float keep = hi ? v[k + O] : v[k];
    if constexpr (O < 16) v[k] = keep + xor_lane<O>(send);
    else v[k] = keep + __shfl_xor(send, O, kWave);
  }
}
__device__ __forceinline__ float transpose_reduce64(float* v, int lane) {
  transpose_reduce_step<32>(v, lane);
  transpose_reduce_step<16>(v, lane);
  transpose_reduce_step<8>(v, lane);
  transpose_reduce_step<4>(v, lane);
  transpose_reduce_step<2>(v, lane);
  transpose_reduce_step<1>(v, lane);
  return v[0];
}

// Batch of a small pool from the responsibility block sums (one whole wave):
// scores summed in block order, top-b by (score desc, index asc).  Leaves
// the pool in pool_s and the chosen source indices, ascending, in bidx.
__device__ void small_batch(const Shape& sh, const Ws& ws, int p, int psize, int bsize, int nblk,
                            int* pool_s, uint32_t* keys, int* chosen, int* bidx, float* scores) {
  const int lane = threadIdx.x & 63;
  pool_s[lane] = (lane < psize) ? ws.pool[p * ws.s_pool + lane] : 0;
  const float* sp = ws.spart + p * ws.s_spart;
  float s = 0.f;
  int b = 0;
  for (; b + 8 <= nblk; b += 8) {
    float t[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) t[q] = sp[static_cast<long long>(b + q) * 64 + lane];
#pragma unroll
    for (int q = 0; q < 8; ++q) s += t[q];
  }
  for (; b < nblk; ++b) s += sp[static_cast<long long>(b) * 64 + lane];
  if (scores && lane < sh.pool_cap) scores[lane] = lane < psize ? s : 0.f;
  keys[lane] = score_key(s);
  __builtin_amdgcn_wave_barrier();
  wave_topb(keys, psize, bsize, chosen);
  __builtin_amdgcn_wave_barrier();
  if (lane < bsize) bidx[lane] = pool_s[chosen[lane]];
}

// Small pools, fused round: (1) the previous round's batch from the
// responsibility sums, recorded by block 0; (2) the coverage refresh
// b_m <- max(b_m, max_{j in batch} Cbar_mj) for every row, into LDS (block 0
// also stores it; a block that reads an already refreshed b_m recomputes the
// same value, since max(b_new, Cbar_mB) = b_new); (3) singleton gains of the
// block's tokens; (4) last block: the pool of this round, excluding the
// selected set and the batch just chosen.
template <bool kGlobalKeys>
__global__ void __launch_bounds__(256)
gains_fused_kernel(Shape sh, Ws ws, int round, int psize, int prev_psize, int prev_bsize, int prev_base,
                   SelOut so) {
  extern __shared__ float dyn[];      // refreshed coverage [ldM], then LDS keys [N]
  __shared__ int hist[512], scan[16], bc[2], flag;
  __shared__ int pool_s[64], chosen[64], bidx[64];
  __shared__ __attribute__((aligned(16))) uint32_t bkeys[64];
  const int p = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  float* bnew = dyn;
  const float* alpha = ws.alpha + p * ws.s_m;
  float* cov = ws.cov + p * ws.s_cov;
  const float* E = ws.E + p * ws.s_E;
  const int nb = round > 0 ? prev_bsize : 0;
  if (round > 0) {
    float* sc = (so.scores && blockIdx.x == 0)
                    ? so.scores + (static_cast<long long>(p) * sh.rounds + round - 1) * sh.pool_cap : nullptr;
    if (wave == 0)
      small_batch(sh, ws, p, prev_psize, prev_bsize, (sh.m + 255) / 256, pool_s, bkeys, chosen, bidx, sc);
    __syncthreads();
    if (blockIdx.x == 0) commit_batch(sh, ws, p, round - 1, prev_bsize, prev_base, pool_s, chosen, so.batch);
    // two row chunks per trip, all their batch-column loads in flight together
    for (int m0 = tid * 4; m0 < sh.m; m0 += 2048) {
      float4 c[2], a[2], b[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int m = min(m0 + h * 1024, sh.ldM - 4);
        a[h] = *reinterpret_cast<const float4*>(alpha + m);
        b[h] = *reinterpret_cast<const float4*>(cov + m);
        c[h] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
      for (int k0 = 0; k0 < nb; k0 += 16) {
        // indices past the batch repeat its last column: a maximum is unchanged
        float4 v[2][16];
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int q = 0; q < 16; ++q)
            v[h][q] = *reinterpret_cast<const float4*>(
                E + static_cast<long long>(bidx[min(k0 + q, nb - 1)]) * sh.ldM + min(m0 + h * 1024, sh.ldM - 4));
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int q = 0; q < 16; ++q) {
            c[h].x = fmaxf(c[h].x, a[h].x * v[h][q].x); c[h].y = fmaxf(c[h].y, a[h].y * v[h][q].y);
            c[h].z = fmaxf(c[h].z, a[h].z * v[h][q].z); c[h].w = fmaxf(c[h].w, a[h].w * v[h][q].w);
          }
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int m = m0 + h * 1024;
        if (m < sh.m) {
          const float4 r = make_float4(fmaxf(b[h].x, c[h].x), fmaxf(b[h].y, c[h].y), fmaxf(b[h].z, c[h].z),
                                       fmaxf(b[h].w, c[h].w));
          *reinterpret_cast<float4*>(bnew + m) = r;
          if (blockIdx.x == 0) *reinterpret_cast<float4*>(cov + m) = r;
        }
      }
    }
  } else {
    // the coverage before the first round: zero, or the image seeds' b_m(S_0)
    for (int m = tid * 4; m < sh.m; m += 1024)
      *reinterpret_cast<float4*>(bnew + m) =
          sh.nseed > 0 ? *reinterpret_cast<const float4*>(cov + m) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  __syncthreads();
  const int col0 = blockIdx.x * kGainColsF + wave * kCpwF;
  float* u = ws.u + p * ws.s_u;
  float acc[kCpwF];
  const float* col[kCpwF];
#pragma unroll
  for (int c = 0; c < kCpwF; ++c) {
    acc[c] = 0.f;
    col[c] = E + static_cast<long long>(min(col0 + c, sh.N - 1)) * sh.ldM;
  }
#pragma unroll 4
  for (int m = lane * 4; m < sh.m; m += 256) {
    const float4 a = *reinterpret_cast<const float4*>(alpha + m);
    const float4 b = *reinterpret_cast<const float4*>(bnew + m);
#pragma unroll
    for (int c = 0; c < kCpwF; ++c) {
      const float4 v = *reinterpret_cast<const float4*>(col[c] + m);
      acc[c] += fmaxf(a.x * v.x - b.x, 0.f);
      acc[c] += fmaxf(a.y * v.y - b.y, 0.f);
      acc[c] += fmaxf(a.z * v.z - b.z, 0.f);
      acc[c] += fmaxf(a.w * v.w - b.w, 0.f);
    }
  }
#pragma unroll
  for (int c = 0; c < kCpwF; ++c) {
    const float s = wave_sum(acc[c]);
    if (lane == 0 && col0 + c < sh.N) st_dev(&u[col0 + c], s);
  }

  int* cnt = ws.cnt + p * ws.s_cnt;
  if (!last_arrival(&cnt[0], gridDim.x, &flag)) return;
  if (tid == 0) st_dev(&cnt[0], 0);
  uint32_t* keys = kGlobalKeys ? ws.keys + p * ws.s_keys : reinterpret_cast<uint32_t*>(dyn + sh.ldM);
  const int* sel = ws.sel + p * ws.s_sel;
  for (int base = 0; base < sh.N; base += 256 * 16) {
    float g[16];
    int sl[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int i = min(base + q * 256 + tid, sh.N - 1);
      g[q] = ld_dev(&u[i]);
      sl[q] = sel[i];
    }
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int i = base + q * 256 + tid;
      if (i < sh.N) {
        bool taken = sl[q] >= 0;
        for (int k = 0; k < nb; ++k) taken |= bidx[k] == i;
        keys[i] = taken ? 0u : score_key(g[q]);
        if (so.gains) so.gains[(static_cast<long long>(p) * sh.rounds + round) * sh.N + i] = taken ? 0.f : g[q];
      }
    }
  }
  __syncthreads();
  int* pool = ws.pool + p * ws.s_pool;
  block_topk256(keys, sh.N, psize, pool, hist, scan, bc);
  if (so.pool) {
    int32_t* tp = so.pool + (static_cast<long long>(p) * sh.rounds + round) * sh.pool_cap;
    for (int j = tid; j < sh.pool_cap; j += 256) tp[j] = (j < psize) ? pool[j] : -1;
  }
}

// Small pools, after the last round: its batch from the responsibility sums.
__global__ void __launch_bounds__(64) final_batch_kernel(Shape sh, Ws ws, int round, int psize, int bsize,
                                                         int sel_base, SelOut so) {
  __shared__ int pool_s[64], chosen[64], bidx[64];
  __shared__ __attribute__((aligned(16))) uint32_t keys[64];
  const int p = blockIdx.x;
  small_batch(sh, ws, p, psize, bsize, (sh.m + 255) / 256, pool_s, keys, chosen, bidx,
              so.scores ? so.scores + (static_cast<long long>(p) * sh.rounds + round) * sh.pool_cap : nullptr);
  __syncthreads();
  commit_batch(sh, ws, p, round, bsize, sel_base, pool_s, chosen, so.batch);
}

// Pool of at most 64: per-block responsibility sums; the batch is picked by
// the next kernel (the next round's gains, or the final batch kernel).
__global__ void __launch_bounds__(256) resp_small_kernel(Shape sh, Params pr, Ws ws, int psize) {
  __shared__ int pool_s[64];
  __shared__ float wsum[4][64];
  const int p = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid < 64) pool_s[tid] = (tid < psize) ? ws.pool[p * ws.s_pool + tid] : 0;
  __syncthreads();
  const int m = blockIdx.x * 256 + tid;
  const bool row_ok = m < sh.m;
  const int mc = row_ok ? m : 0;   // clamped: every load below is unconditional
  const float* E = ws.E + p * ws.s_E + mc;
  float v[64];
  float mu = 0.f;
  const float a = row_ok ? ws.alpha[p * ws.s_m + mc] : 0.f;
  const float c = ws.cov[p * ws.s_cov + mc];
#pragma unroll
  for (int j = 0; j < 64; ++j) v[j] = E[static_cast<long long>(pool_s[j]) * sh.ldM];
#pragma unroll
  for (int j = 0; j < 64; ++j) {
    const float r = (j < psize) ? fmaxf(a * v[j] - c, 0.f) : 0.f;
    v[j] = r;
    mu = fmaxf(mu, r);
  }
  if (mu > 0.f) {
    const float inv = 1.f / (pr.tau_r * mu + pr.resp_eps);
    const float zmax = mu * inv;
    float den = 0.f;
    float ex[64];
#pragma unroll
    for (int j = 0; j < 64; ++j) {
      ex[j] = (j < psize) ? __expf(v[j] * inv - zmax) : 0.f;
      den += ex[j];
    }
    const float rden = 1.f / den;
#pragma unroll
    for (int j = 0; j < 64; ++j) v[j] = ex[j] * rden * v[j];
  } else {
#pragma unroll
    for (int j = 0; j < 64; ++j) v[j] = 0.f;
  }
  wsum[wave][lane] = transpose_reduce64(v, lane);
  __syncthreads();
  float* sp = ws.spart + p * ws.s_spart;
  if (tid < psize)
    sp[static_cast<long long>(blockIdx.x) * 64 + tid] = ((wsum[0][tid] + wsum[1][tid]) + wsum[2][tid]) + wsum[3][tid];
}

// Large pools: per-row max mu_m and softmax denominator over the pool.
// Block = 64 rows (lane = row) x 16 waves splitting the pool positions (the
// grid is only m / 64 blocks, so the waves supply the loads in flight).
constexpr int kRsW = 16;
__global__ void __launch_bounds__(64 * kRsW) rowstat_kernel(Shape sh, Params pr, Ws ws, int psize) {
  __shared__ float part[kRsW][64];
  __shared__ float mu_s[64];
  const int p = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int m = blockIdx.x * 64 + lane;
  const bool row_ok = m < sh.m;
  const float a = row_ok ? ws.alpha[p * ws.s_m + m] : 0.f;
  const float c = row_ok ? ws.cov[p * ws.s_cov + m] : 0.f;
  const float* E = ws.E + p * ws.s_E + (row_ok ? m : 0);
  const int* pool = ws.pool + p * ws.s_pool;
  const int q = (psize + kRsW - 1) / kRsW, j0 = wave * q, j1 = min(psize, j0 + q);
  float mx = 0.f;
#pragma unroll 32
  for (int j = j0; j < j1; ++j) mx = fmaxf(mx, fmaxf(a * E[static_cast<long long>(pool[j]) * sh.ldM] - c, 0.f));
  part[wave][lane] = mx;
  __syncthreads();
  if (wave == 0) {
    float mm = part[0][lane];
#pragma unroll
    for (int w = 1; w < kRsW; ++w) mm = fmaxf(mm, part[w][lane]);
    mu_s[lane] = mm;
  }
  __syncthreads();
  const float mu = mu_s[lane];
  const float inv = mu > 0.f ? 1.f / (pr.tau_r * mu + pr.resp_eps) : 0.f;
  const float zmax = mu * inv;
  float den = 0.f;
  if (mu > 0.f)
#pragma unroll 32
    for (int j = j0; j < j1; ++j)
      den += __expf(fmaxf(a * E[static_cast<long long>(pool[j]) * sh.ldM] - c, 0.f) * inv - zmax);
  __syncthreads();
  part[wave][lane] = den;
  __syncthreads();
  if (wave == 0 && row_ok) {
    float d = part[0][lane];
#pragma unroll
    for (int w = 1; w < kRsW; ++w) d += part[w][lane];
    float* rs = ws.rstat + p * ws.s_rstat;
    rs[m] = inv;
    rs[sh.ldM + m] = zmax;
    rs[2 * sh.ldM + m] = mu > 0.f ? 1.f / d : 0.f;
  }
}

// Large pools: one wave per pool position sums rho R over all client rows;
// the last block picks the batch.
__global__ void __launch_bounds__(256)
colsum_kernel(Shape sh, Ws ws, int round, int psize, int bsize, int sel_base, SelOut so) {
  extern __shared__ uint32_t keys[];   // pool_cap words
  __shared__ int hist[512], scan[16], bc[2], flag;
  __shared__ int chosen[1024];
  const int p = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int jj = blockIdx.x * 4 + wave;
  const int* pool = ws.pool + p * ws.s_pool;
  const float* rs = ws.rstat + p * ws.s_rstat;
  const float* alpha = ws.alpha + p * ws.s_m;
  const float* cov = ws.cov + p * ws.s_cov;
  float* sv = ws.u + p * ws.s_u;        // scores reuse the gains buffer
  if (jj < psize) {
    const float* col = ws.E + p * ws.s_E + static_cast<long long>(pool[jj]) * sh.ldM;
    float acc = 0.f;
    for (int m = lane * 4; m < sh.m; m += 256) {
      const float4 v = *reinterpret_cast<const float4*>(col + m);
      const float4 a = *reinterpret_cast<const float4*>(alpha + m);
      const float4 c = *reinterpret_cast<const float4*>(cov + m);
      const float4 inv = *reinterpret_cast<const float4*>(rs + m);
      const float4 zm = *reinterpret_cast<const float4*>(rs + sh.ldM + m);
      const float4 rd = *reinterpret_cast<const float4*>(rs + 2 * sh.ldM + m);
      float r;
      r = fmaxf(a.x * v.x - c.x, 0.f); acc += __expf(r * inv.x - zm.x) * rd.x * r;
      r = fmaxf(a.y * v.y - c.y, 0.f); acc += __expf(r * inv.y - zm.y) * rd.y * r;
      r = fmaxf(a.z * v.z - c.z, 0.f); acc += __expf(r * inv.z - zm.z) * rd.z * r;
      r = fmaxf(a.w * v.w - c.w, 0.f); acc += __expf(r * inv.w - zm.w) * rd.w * r;
    }
    const float s = wave_sum(acc);
    if (lane == 0) st_dev(&sv[jj], s);
  }
  int* cnt = ws.cnt + p * ws.s_cnt;
  if (!last_arrival(&cnt[4], gridDim.x, &flag)) return;
  if (tid == 0) st_dev(&cnt[4], 0);
  {
    float g[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) g[q] = ld_dev(&sv[min(q * 256 + tid, psize - 1)]);
#pragma unroll
    for (int q = 0; q < 8; ++q)
      if (q * 256 + tid < psize) keys[q * 256 + tid] = score_key(g[q]);
    if (so.scores) {
      float* sc = so.scores + (static_cast<long long>(p) * sh.rounds + round) * sh.pool_cap;
#pragma unroll
      for (int q = 0; q < 8; ++q)
        if (q * 256 + tid < sh.pool_cap) sc[q * 256 + tid] = q * 256 + tid < psize ? g[q] : 0.f;
    }
  }
  __syncthreads();
  block_topk256(keys, psize, bsize, chosen, hist, scan, bc);
  commit_batch(sh, ws, p, round, bsize, sel_base, pool, chosen, so.batch);
}

// ---------------------------------------------------------------------------
// Persistent selection: every round of a small-pool call in one launch.  The
// grid is nblk blocks per problem, sized to be co-resident (one block per CU,
// two for the streamed kernel when it fits twice); every block keeps its own
// copy of the coverage b_m in LDS and reads the row weights from L2.  A round:
//   gains  - waves stream the client rows of unselected tokens (round robin
//            over all waves of the problem) and publish u_i tagged with the
//            round number
//   pool   - every block that owns a row chunk (and the last block) waits
//            for the tagged gains and picks the same pool (identical inputs,
//            deterministic top-k)
//   resp   - one block per 64-row chunk, its waves splitting the pool:
//            responsibility softmax over the pool, per-chunk sums per pool
//            token, published tagged
//   batch  - those blocks wait for the tagged chunk sums, add them in chunk
//            order and pick the same batch; the last block records it and
//            block 0 publishes its tokens, which are all the other blocks
//            wait for (with one chunk per block)
//   cov    - one wave per 64-row chunk: b_m <- max(b_m, max_{j in batch}
//            Cbar_mj), published tagged; every block waits for the tags and
//            copies b into LDS
// In the last round only the last block continues after the batch: it
// refreshes its own coverage copy, writes the coverage, F(S) and F(V), and
// the support list (ascending, with each token's slot).
//
// Tagged values are double-buffered by round parity, so a buffer is rewritten
// two rounds after the round that read it.  Along with its coverage rows each
// block publishes a tagged heartbeat (after it has read everything of the
// round except the coverage; a block without the pool reads only the batch's
// tokens, whose slots are rewritten only after every block's gains two
// rounds on, so it publishes first), and the coverage hand-off waits for
// every block's heartbeat as well as for the rows.  A block therefore starts round
// r + 1 only after every block has finished its reads of round r - 1 and
// earlier, so no value is overwritten before all its readers are done; the
// ordering rides on a poll that happens anyway, with no barrier and no
// same-address atomics.  Every wait is
// bounded: after kSpinLimit polls, or once this block has recorded a timeout,
// the block records the timeout (device status word) and stops waiting, so
// every wave always exits.
constexpr int kSpinLimit = 1 << 18;   // bounded waits (a fraction of a second)

// Marks the call failed (sticky device status bit) after a bounded wait.
__device__ __forceinline__ void mark_timeout(int* cnt, int* failed) {
  raise_status(cnt, kStatusSelect);
  *failed = 1;
}

// Entry i of the coverage hand-off poll: rows [0, m), then the heartbeats at
// [ldM, ldM + nblk); the padding rows [m, ldM) are never written and poll
// row m - 1 instead.
__device__ __forceinline__ int stage_index(int i, const Shape& sh, int nst) {
  i = min(i, nst - 1);
  return (i >= sh.m && i < sh.ldM) ? sh.m - 1 : i;
}

// Pool of the persistent selection with the keys in registers: thread t
// takes the gains of its contiguous segment (taken tokens key 0), waiting
// until each carries this round's tag.
template <int KPT>
__device__ __forceinline__ void pool_regs(const Shape& sh, const unsigned long long* tu, unsigned tag,
                                          const unsigned char* taken, int psize, int* pool_s, int* hist, int* scan,
                                          int* cnt, int* failed) {
  const int seg = (sh.N + 255) / 256;
  const int i0 = threadIdx.x * seg;
  unsigned long long w[KPT];
  bool need[KPT];
#pragma unroll
  for (int q = 0; q < KPT; ++q) {
    const int i = min(i0 + q, sh.N - 1);
    need[q] = q < seg && i0 + q < sh.N && !taken[i];
    w[q] = ld_dev64(&tu[i]);
  }
  for (int spin = 0;; ++spin) {
    bool pend = false;
#pragma unroll
    for (int q = 0; q < KPT; ++q) pend |= need[q] && tag_of(w[q]) != tag;
    if (!pend || *failed) break;
    if (spin == kSpinLimit) { mark_timeout(cnt, failed); break; }
    __builtin_amdgcn_s_sleep(1);
#pragma unroll
    for (int q = 0; q < KPT; ++q)
      if (need[q] && tag_of(w[q]) != tag) w[q] = ld_dev64(&tu[min(i0 + q, sh.N - 1)]);
  }
  uint32_t k[KPT];
#pragma unroll
  for (int q = 0; q < KPT; ++q) k[q] = need[q] ? score_key(value_of(w[q])) : 0u;
  block_topk_regs<KPT>(k, seg, psize, pool_s, hist, scan);
}

// A wave-uniform value the compiler cannot see through (so it is not
// hoisted out of a loop): through a VGPR and back.
__device__ __forceinline__ int opaque_uniform(int v) {
  asm volatile("" : "+v"(v));
  return __builtin_amdgcn_readfirstlane(v);
}

// RES: block b owns tokens [8 b, 8 b + 8) (N <= 8 blocks, M <= 256 kResJ) and
// keeps their weighted client rows alpha_m E[i][m] (Cbar, the product rounded
// once) in registers for the whole call, wave w holding the rows
// m = 64 (w + 4 j) + lane, j < kResJ, of all eight tokens; a round's gains
// then read only the coverage.  Otherwise each wave streams the rows of
// its tokens (gw, gw + waves, ...) from the caches every round.
constexpr int kResJ = 14;
template <bool RES>
__global__ void __launch_bounds__(256)
select_persistent_kernel(Shape sh, Params pr, Ws ws, int nblk, SelOut so, int quad) {
  extern __shared__ float dyn[];
  // LDS: b_m [ldM] | selected flags [N, padded to 16 bytes] | pool keys [N]
  //      (only when N exceeds the register top-k); the row weights are read
  //      from L2 beside the client values they scale, which keeps a block
  //      small enough for two per CU on the document page
  float* bl = dyn;
  unsigned char* taken = reinterpret_cast<unsigned char*>(dyn + sh.ldM);
  uint32_t* keys = reinterpret_cast<uint32_t*>(taken + ((sh.N + 15) & ~15));
  __shared__ int hist[768], scan[16], bc[2], failed;
  __shared__ int pool_s[64], chosen[64], bidx[64];
  __shared__ __attribute__((aligned(16))) uint32_t bkeys[64];
  __shared__ float rmu[4][64], rden_s[4][64], red[16];
  // Cbar of the chunk's rows at the pool's tokens (pool position, row lane),
  // kept from the responsibilities for the coverage refresh
  __shared__ float cpool[64][64];
  const int p = blockIdx.y, blk = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nwaves = nblk * 4, gw = blk * 4 + wave;
  const int nchunk = (sh.m + 63) / 64;
  // the pool and the chunk sums are needed by the blocks that own a row
  // chunk (responsibilities, coverage) and by the last block (it records the
  // batch); with one chunk per block the others skip both and wait only for
  // the batch's tokens, which block 0 publishes after its pick
  const bool pool_here = nchunk > nblk || blk < nchunk || blk == nblk - 1;
  const bool pool_pub = nchunk + 1 < nblk;
  const float* E = ws.E + p * ws.s_E;
  unsigned long long* tu = ws.tu + p * ws.s_tu;
  unsigned long long* ts = ws.ts + p * ws.s_ts;
  unsigned long long* tc = ws.tc + p * ws.s_tc;
  const float* alpha_g = ws.alpha + p * ws.s_m;
  int* cnt = ws.cnt + p * ws.s_cnt;
  {
    const float* cov0 = ws.cov + p * ws.s_cov;
    for (int m = tid; m < sh.ldM; m += 256) {
      // coverage at the first round: zero, or the image seeds' b_m(S_0)
      bl[m] = sh.nseed > 0 ? cov0[m] : 0.f;
    }
  }
  {
    const int* sel0 = ws.sel + p * ws.s_sel;
    for (int i = tid; i < sh.N; i += 256) taken[i] = (sh.nseed > 0 && sel0[i] >= 0) ? 1 : 0;
  }
  if (tid == 0) failed = 0;
  float er[RES ? 8 : 1][RES ? kResJ : 1];
  if constexpr (RES) {
    // rows past M and tokens past N hold zeros (clamped loads, then select)
#pragma unroll
    for (int j = 0; j < kResJ; ++j) {
      const int m = 64 * (wave + 4 * j) + lane;
      const int mc = min(m, sh.m - 1);
      const float a = alpha_g[mc];
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const int t = blk * 8 + s;
        const float v = E[static_cast<long long>(min(t, sh.N - 1)) * sh.ldM + mc];
        er[s][j] = (m < sh.m && t < sh.N) ? a * v : 0.f;
      }
    }
  }
  __syncthreads();
  int selected = sh.nseed;
  const Shape sh_call = sh;
  const int tid_call = tid;
  for (int r = 0; r < sh_call.rounds; ++r) {
    // Opaque per-round copies of the shape and the thread index: index math
    // derived from them is redone every round instead of being hoisted out
    // of the loop and kept live (in spill registers) across all rounds.
    Shape sh = sh_call;
    int tid = tid_call;
    sh.N = opaque_uniform(sh.N);
    sh.m = opaque_uniform(sh.m);
    sh.ldM = opaque_uniform(sh.ldM);
    sh.K = opaque_uniform(sh.K);
    sh.b = opaque_uniform(sh.b);
    sh.pool_cap = opaque_uniform(sh.pool_cap);
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63, wave = tid >> 6, gw = blk * 4 + wave;
    const int psize = min(sh.pool_cap, sh.N - selected);
    const int bsize = min(sh.b, sh.K - selected);
    const unsigned tag = static_cast<unsigned>(r + 1);
    unsigned long long* tur = tu + (r & 1) * sh.N;
    unsigned long long* tsr = ts + (r & 1) * 64LL * nchunk;

    // ---- singleton gains of unselected tokens, two tokens per wave pass with
    //      all their row loads in flight (or the block's rows held in registers),
    //      published with this round's tag
    if constexpr (RES) {
      // per lane: the partial gains of the eight tokens over its rows
      // (b_m >= 0, so rows past M add zero); then summed over the lanes and
      // the four waves, in that order
      float acc[8];
#pragma unroll
      for (int s = 0; s < 8; ++s) acc[s] = 0.f;
#pragma unroll
      for (int j = 0; j < kResJ; ++j) {
        const float b = bl[min(64 * (wave + 4 * j) + lane, sh.ldM - 1)];
#pragma unroll
        for (int s = 0; s < 8; ++s) acc[s] += fmaxf(er[s][j] - b, 0.f);
      }
      transpose_reduce_step<4>(acc, lane);
      transpose_reduce_step<2>(acc, lane);
      transpose_reduce_step<1>(acc, lane);
      float g = acc[0];             // token lane & 7, summed over 8 lanes
      g += xor_lane<8>(g);
      g = add_xor16(g);
      g = add_xor32(g);
      if (lane < 8) rmu[wave][lane] = g;
      __syncthreads();
      if (tid < 8) {
        const int t = blk * 8 + tid;
        const float g = ((rmu[0][tid] + rmu[1][tid]) + rmu[2][tid]) + rmu[3][tid];
        if (t < sh.N && !taken[t]) st_dev64(&tur[t], tag_value(tag, g));
        if (so.gains && t < sh.N)
          so.gains[(static_cast<long long>(p) * sh.rounds + r) * sh.N + t] = taken[t] ? 0.f : g;
      }
    } else if (quad) {
      // one block per CU: four tokens per wave pass, all their row loads in
      // flight together (each token's sum is formed exactly as in the
      // two-token loop below)
      for (int i0 = gw; i0 < sh.N; i0 += 4 * nwaves) {
        int it[4];
        bool ok[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          it[k] = i0 + k * nwaves;
          ok[k] = it[k] < sh.N && taken[min(it[k], sh.N - 1)] == 0;
        }
        float* gout = so.gains ? so.gains + (static_cast<long long>(p) * sh.rounds + r) * sh.N : nullptr;
        if (!(ok[0] || ok[1] || ok[2] || ok[3])) {
          if (gout && lane == 0)
#pragma unroll
            for (int k = 0; k < 4; ++k)
              if (it[k] < sh.N) gout[it[k]] = 0.f;
          continue;
        }
        // a token that needs no gain re-reads a needed one's row (cache hits)
        const int any = ok[0] ? it[0] : ok[1] ? it[1] : ok[2] ? it[2] : it[3];
        const float* c[4];
        float acc[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          c[k] = E + static_cast<long long>(ok[k] ? it[k] : any) * sh.ldM;
          acc[k] = 0.f;
        }
#pragma unroll 4
        for (int m = lane * 4; m < sh.m; m += 256) {
          const float4 a = *reinterpret_cast<const float4*>(alpha_g + m);
          const float4 b = *reinterpret_cast<const float4*>(bl + m);
          float4 v[4];
#pragma unroll
          for (int k = 0; k < 4; ++k) v[k] = *reinterpret_cast<const float4*>(c[k] + m);
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            acc[k] += fmaxf(a.x * v[k].x - b.x, 0.f); acc[k] += fmaxf(a.y * v[k].y - b.y, 0.f);
            acc[k] += fmaxf(a.z * v[k].z - b.z, 0.f); acc[k] += fmaxf(a.w * v[k].w - b.w, 0.f);
          }
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) acc[k] = wave_sum(acc[k]);
        if (lane == 0)
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            if (ok[k]) st_dev64(&tur[it[k]], tag_value(tag, acc[k]));
            if (gout && it[k] < sh.N) gout[it[k]] = ok[k] ? acc[k] : 0.f;
          }
      }
    } else
    for (int i0 = gw; i0 < sh.N; i0 += 2 * nwaves) {
      const int i1 = i0 + nwaves;
      const bool ok0 = taken[i0] == 0;
      const bool ok1 = i1 < sh.N && taken[min(i1, sh.N - 1)] == 0;
      float* gout = so.gains ? so.gains + (static_cast<long long>(p) * sh.rounds + r) * sh.N : nullptr;
      if (!ok0 && !ok1) {
        if (gout && lane == 0) {
          gout[i0] = 0.f;
          if (i1 < sh.N) gout[i1] = 0.f;
        }
        continue;
      }
      // a token that needs no gain re-reads the other one's row (cache hits)
      const float* c0 = E + static_cast<long long>(ok0 ? i0 : i1) * sh.ldM;
      const float* c1 = E + static_cast<long long>(ok1 ? i1 : i0) * sh.ldM;
      float a0 = 0.f, a1 = 0.f;
#pragma unroll 4
      for (int m = lane * 4; m < sh.m; m += 256) {
        const float4 a = *reinterpret_cast<const float4*>(alpha_g + m);
        const float4 b = *reinterpret_cast<const float4*>(bl + m);
        const float4 v0 = *reinterpret_cast<const float4*>(c0 + m);
        const float4 v1 = *reinterpret_cast<const float4*>(c1 + m);
        a0 += fmaxf(a.x * v0.x - b.x, 0.f); a0 += fmaxf(a.y * v0.y - b.y, 0.f);
        a0 += fmaxf(a.z * v0.z - b.z, 0.f); a0 += fmaxf(a.w * v0.w - b.w, 0.f);
        a1 += fmaxf(a.x * v1.x - b.x, 0.f); a1 += fmaxf(a.y * v1.y - b.y, 0.f);
        a1 += fmaxf(a.z * v1.z - b.z, 0.f); a1 += fmaxf(a.w * v1.w - b.w, 0.f);
      }
      a0 = wave_sum(a0);
      a1 = wave_sum(a1);
      if (lane == 0) {
        if (ok0) st_dev64(&tur[i0], tag_value(tag, a0));
        if (ok1) st_dev64(&tur[i1], tag_value(tag, a1));
        if (gout) {
          gout[i0] = ok0 ? a0 : 0.f;
          if (i1 < sh.N) gout[i1] = ok1 ? a1 : 0.f;
        }
      }
    }

    // ---- the pool, identical in every block that needs it (waits for this
    //      round's gains)
    // the batch's tokens, published by block 0 for the blocks without the pool
    unsigned long long* tpr = ts + 128LL * nchunk + (r & 1) * 64;
    if (pool_here) {
    if constexpr (RES) {
      if (sh.N <= 256 * 6)
        pool_regs<6>(sh, tur, tag, taken, psize, pool_s, hist, scan, cnt, &failed);
      else
        pool_regs<8>(sh, tur, tag, taken, psize, pool_s, hist, scan, cnt, &failed);
    } else if (sh.N <= 256 * 8)
      pool_regs<8>(sh, tur, tag, taken, psize, pool_s, hist, scan, cnt, &failed);
    else if (sh.N <= 256 * 16)
      pool_regs<16>(sh, tur, tag, taken, psize, pool_s, hist, scan, cnt, &failed);
    else {
      for (int base = 0; base < sh.N; base += 256 * 16) {
        unsigned long long w[16];
        bool need[16];
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int i = base + q * 256 + tid;
          need[q] = i < sh.N && !taken[min(i, sh.N - 1)];
          w[q] = ld_dev64(&tur[min(i, sh.N - 1)]);
        }
        for (int spin = 0;; ++spin) {
          bool pend = false;
#pragma unroll
          for (int q = 0; q < 16; ++q) pend |= need[q] && tag_of(w[q]) != tag;
          if (!pend || failed) break;
          if (spin == kSpinLimit) { mark_timeout(cnt, &failed); break; }
          __builtin_amdgcn_s_sleep(1);
#pragma unroll
          for (int q = 0; q < 16; ++q)
            if (need[q] && tag_of(w[q]) != tag) w[q] = ld_dev64(&tur[min(base + q * 256 + tid, sh.N - 1)]);
        }
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int i = base + q * 256 + tid;
          if (i < sh.N) keys[i] = need[q] ? score_key(value_of(w[q])) : 0u;
        }
      }
      __syncthreads();
      block_topk256(keys, sh.N, psize, pool_s, hist, scan, bc);
    }
    if constexpr (!RES) {
      // clamp to valid rows (defensive) and pad past psize with a valid row,
      // masked below (the register top-k pads with row 0 itself)
      int pv = 0;
      if (tid < 64) pv = min(max(pool_s[tid < psize ? tid : 0], 0), sh.N - 1);
      __syncthreads();
      if (tid < 64) pool_s[tid] = pv;
      __syncthreads();
    }
    }
    if (blk == nblk - 1 && so.pool) {
      int32_t* tp = so.pool + (static_cast<long long>(p) * sh.rounds + r) * sh.pool_cap;
      for (int j = tid; j < sh.pool_cap; j += 256) tp[j] = (j < psize) ? pool_s[j] : -1;
    }

    // ---- responsibilities: one block per 64-row chunk (lane = client row),
    //      its four waves split the pool positions 16 apiece; the per-chunk
    //      sums are published with this round's tag
    for (int c = blk; c < nchunk; c += nblk) {
      const int m = c * 64 + lane;
      const bool row_ok = m < sh.m;
      const int mc = row_ok ? m : 0;
      const float a = row_ok ? alpha_g[mc] : 0.f;
      const float b = bl[mc];
      const int j0 = wave * 16;
      float v[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) v[j] = E[static_cast<long long>(pool_s[j0 + j]) * sh.ldM + mc];
      float mu = 0.f;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const float cb = a * v[j];
        cpool[j0 + j][lane] = cb;
        const float rr = (j0 + j < psize) ? fmaxf(cb - b, 0.f) : 0.f;
        v[j] = rr;
        mu = fmaxf(mu, rr);
      }
      rmu[wave][lane] = mu;
      __syncthreads();
      mu = fmaxf(fmaxf(rmu[0][lane], rmu[1][lane]), fmaxf(rmu[2][lane], rmu[3][lane]));
      const float inv = mu > 0.f ? 1.f / (pr.tau_r * mu + pr.resp_eps) : 0.f;
      const float zmax = mu * inv;
      float den = 0.f;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const float ex = (j0 + j < psize) ? __expf(v[j] * inv - zmax) : 0.f;
        den += ex;
        v[j] *= ex;    // rho numerator times R; scaled by 1/den below
      }
      rden_s[wave][lane] = den;
      __syncthreads();
      den = ((rden_s[0][lane] + rden_s[1][lane]) + rden_s[2][lane]) + rden_s[3][lane];
      const float rden = mu > 0.f ? 1.f / den : 0.f;
#pragma unroll
      for (int j = 0; j < 16; ++j) v[j] *= rden;
      // sum over the 64 rows per pool position: butterfly inside 16-lane
      // groups, then across the four groups
      transpose_reduce_step<8>(v, lane);
      transpose_reduce_step<4>(v, lane);
      transpose_reduce_step<2>(v, lane);
      transpose_reduce_step<1>(v, lane);
      float tot = v[0];
      tot = add_xor16(tot);
      tot = add_xor32(tot);
      if (lane < 16) st_dev64(&tsr[static_cast<long long>(c) * 64 + j0 + lane], tag_value(tag, tot));
      __syncthreads();   // rmu / rden_s are reused by the next chunk
    }

    // ---- the batch, identical in every block with the pool: each wave waits
    //      for the tagged sums of a quarter of the chunks (16 loads in
    //      flight) and adds them in chunk order; the quarters are added in
    //      wave order.  The other blocks wait for the batch's tokens alone.
    if (!pool_here) {
      // nothing left for these blocks in the last round
      if (r + 1 == sh.rounds) break;
      // they read nothing else of this round (the batch's slots are
      // rewritten two rounds on, after every block's gains of that round),
      // so their heartbeat goes out before the wait
      if (tid == 0) st_dev64(&tc[(r & 1) * (sh.ldM + kMaxPersist) + sh.ldM + blk], tag_value(tag, 0.f));
      if (tid < 16) {
        unsigned long long bw = ld_dev64(&tpr[tid]);
        for (int spin = 0; tag_of(bw) != tag && !failed; ++spin) {
          if (spin == kSpinLimit) { mark_timeout(cnt, &failed); break; }
          __builtin_amdgcn_s_sleep(1);
          bw = ld_dev64(&tpr[tid]);
        }
        bidx[tid] = min(max(__float_as_int(value_of(bw)), 0), sh.N - 1);
      }
      __syncthreads();
    } else {
    {
      const int per = (nchunk + 3) / 4;
      const int c_end = min(nchunk, (wave + 1) * per);
      float s = 0.f;
      for (int c0 = wave * per; c0 < c_end; c0 += 16) {
        unsigned long long w[16];
#pragma unroll
        for (int q = 0; q < 16; ++q) w[q] = ld_dev64(&tsr[static_cast<long long>(min(c0 + q, c_end - 1)) * 64 + lane]);
        for (int spin = 0;; ++spin) {
          bool pend = false;
#pragma unroll
          for (int q = 0; q < 16; ++q) pend |= tag_of(w[q]) != tag;
          if (!pend || failed) break;
          if (spin == kSpinLimit) { mark_timeout(cnt, &failed); break; }
          __builtin_amdgcn_s_sleep(1);
#pragma unroll
          for (int q = 0; q < 16; ++q)
            if (tag_of(w[q]) != tag) w[q] = ld_dev64(&tsr[static_cast<long long>(min(c0 + q, c_end - 1)) * 64 + lane]);
        }
#pragma unroll
        for (int q = 0; q < 16; ++q)
          if (c0 + q < c_end) s += value_of(w[q]);
      }
      rmu[wave][lane] = s;   // free: the responsibility loop ended with a barrier
    }
    __syncthreads();
    if (wave == 0) {
      const float s = ((rmu[0][lane] + rmu[1][lane]) + rmu[2][lane]) + rmu[3][lane];
      if (blk == nblk - 1 && so.scores && lane < sh.pool_cap)
        so.scores[(static_cast<long long>(p) * sh.rounds + r) * sh.pool_cap + lane] = lane < psize ? s : 0.f;
      bkeys[lane] = score_key(s);
      __builtin_amdgcn_wave_barrier();
      wave_topb(bkeys, psize, bsize, chosen);
      __builtin_amdgcn_wave_barrier();
      if (lane < bsize) bidx[lane] = pool_s[chosen[lane]];
      __builtin_amdgcn_wave_barrier();
      if (pool_pub && blk == 0 && lane < 16)
        st_dev64(&tpr[lane], tag_value(tag, __int_as_float(lane < bsize ? bidx[lane] : 0)));
    }
    __syncthreads();
    }
    const bool last = r + 1 == sh.rounds;
    // the last block records the batch (and alone finishes the last round)
    if (blk == nblk - 1) commit_batch(sh, ws, p, r, bsize, selected, pool_s, chosen, so.batch);
    else if (last) break;
    if (tid < bsize) taken[bidx[tid]] = 1;
    if (!last) {
      // ---- coverage refresh with the batch, published with this round's
      //      tag: with one chunk per block, by the chunk's responsibility
      //      block (its pool columns, the batch among them, were just read
      //      here, so the loads hit this XCD's L2), wave w taking batch
      //      entries w, w + 4, ...; otherwise one wave per 64-row chunk
      unsigned long long* tcr = tc + (r & 1) * (sh.ldM + kMaxPersist);
      if (nchunk <= nblk && bsize <= 16) {
        if (blk < nchunk) {
          const int m = blk * 64 + lane;
          const int mc = min(m, sh.m - 1);
          // the pool holds at most 64 = 4 b entries here, so b <= 16: four
          // batch entries per wave, their Cbar values kept in LDS by this
          // block's responsibility pass over the same rows
          float cm = bl[mc];
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (wave + 4 * q < bsize) cm = fmaxf(cm, cpool[chosen[wave + 4 * q]][lane]);
          rmu[wave][lane] = cm;   // free: last read before the barrier after the batch
          __syncthreads();
          if (wave == 0 && m < sh.m)
            st_dev64(&tcr[m], tag_value(tag, fmaxf(fmaxf(rmu[0][lane], rmu[1][lane]), fmaxf(rmu[2][lane], rmu[3][lane]))));
        }
      } else
      for (int c = gw; c < nchunk; c += nwaves) {
        const int m = c * 64 + lane;
        const int mc = min(m, sh.m - 1);
        const float a = alpha_g[mc];
        float cm = bl[mc];
        for (int k0 = 0; k0 < bsize; k0 += 16) {
          float v[16];
#pragma unroll
          for (int q = 0; q < 16; ++q) v[q] = E[static_cast<long long>(bidx[min(k0 + q, bsize - 1)]) * sh.ldM + mc];
#pragma unroll
          for (int q = 0; q < 16; ++q) cm = fmaxf(cm, a * v[q]);
        }
        if (m < sh.m) st_dev64(&tcr[m], tag_value(tag, cm));
      }
      // this block's heartbeat: it has read everything of earlier rounds
      if (pool_here && tid == 0) st_dev64(&tcr[sh.ldM + blk], tag_value(tag, 0.f));
      // ---- every block copies the refreshed coverage into LDS, waiting for
      //      the tags and for every block's heartbeat
      const int nst = sh.ldM + nblk;
      for (int m0 = 0; m0 < nst; m0 += 256 * 16) {
        unsigned long long w[16];
#pragma unroll
        for (int q = 0; q < 16; ++q) w[q] = ld_dev64(&tcr[stage_index(m0 + q * 256 + tid, sh, nst)]);
        for (int spin = 0;; ++spin) {
          bool pend = false;
#pragma unroll
          for (int q = 0; q < 16; ++q) pend |= tag_of(w[q]) != tag;
          if (!pend || failed) break;
          if (spin == kSpinLimit) { mark_timeout(cnt, &failed); break; }
          __builtin_amdgcn_s_sleep(1);
#pragma unroll
          for (int q = 0; q < 16; ++q)
            if (tag_of(w[q]) != tag) w[q] = ld_dev64(&tcr[stage_index(m0 + q * 256 + tid, sh, nst)]);
        }
#pragma unroll
        for (int q = 0; q < 16; ++q)
          if (m0 + q * 256 + tid < sh.m) bl[m0 + q * 256 + tid] = value_of(w[q]);
      }
      __syncthreads();
      selected += bsize;
      continue;
    }

    // ---- the last round (last block only): coverage refresh of the LDS copy
    //      with two row groups per trip, 16 batch rows each, all loads in flight
    for (int m0 = tid * 4; m0 < sh.m; m0 += 2048) {
      float4 c[2];
      c[0] = c[1] = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int k0 = 0; k0 < bsize; k0 += 16) {
        // indices past the batch repeat its last row: a maximum is unchanged
        float4 v[2][16];
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int q = 0; q < 16; ++q)
            v[h][q] = *reinterpret_cast<const float4*>(E + static_cast<long long>(bidx[min(k0 + q, bsize - 1)]) * sh.ldM +
                                                       min(m0 + h * 1024, sh.ldM - 4));
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int q = 0; q < 16; ++q) {
            c[h].x = fmaxf(c[h].x, v[h][q].x); c[h].y = fmaxf(c[h].y, v[h][q].y);
            c[h].z = fmaxf(c[h].z, v[h][q].z); c[h].w = fmaxf(c[h].w, v[h][q].w);
          }
      }
      // alpha_m >= 0, so alpha_m max_j Et[j][m] = max_j Cbar_mj exactly
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int m = m0 + h * 1024;
        if (m < sh.m) {
          const float4 a = *reinterpret_cast<const float4*>(alpha_g + m);
          float4 b = *reinterpret_cast<const float4*>(bl + m);
          b.x = fmaxf(b.x, a.x * c[h].x); b.y = fmaxf(b.y, a.y * c[h].y);
          b.z = fmaxf(b.z, a.z * c[h].z); b.w = fmaxf(b.w, a.w * c[h].w);
          *reinterpret_cast<float4*>(bl + m) = b;
        }
      }
    }
    selected += bsize;
    __syncthreads();
    if (last) {
      // the last block: the coverage, F(S) = sum_m b_m and F(V) = sum_m
      // max_i Cbar_mi, then the support list in ascending source order with
      // each token's slot
      float* cov = ws.cov + p * ws.s_cov;
      const float* peak = ws.peak + p * ws.s_m;
      float fs = 0.f, fv = 0.f;
      for (int m = tid; m < sh.m; m += 256) {
        cov[m] = bl[m];
        fs += bl[m];
        fv += peak[m];
      }
      fs = block_sum(fs, red);
      fv = block_sum(fv, red);
      int* sup = ws.sup + p * ws.s_sup;
      int* slot = ws.slot + p * ws.s_slot;
      int base = 0;
      for (int b0 = 0; b0 < sh.N; b0 += 256) {
        const int i = b0 + tid;
        const int f = (i < sh.N && taken[i]) ? 1 : 0;
        int tot;
        const int pos = base + block_exclusive_scan(f, scan, &tot);
        if (i < sh.N) {
          slot[i] = f ? pos : -1;
          if (f) sup[pos] = i;
        }
        base += tot;
      }
      if (tid == 0) {
        float* st = ws.stats + p * ws.s_st;
        st[2] = fs;
        st[3] = fv;
        st[4] = static_cast<float>(sh.K);
        st[5] = static_cast<float>(sh.rounds);
        st[6] = static_cast<float>(sh.m);
        st[7] = static_cast<float>(sh.N - sh.K);
      }
      break;
    }
  }
}

// F(S) = sum_m b_m(S) and F(V) = sum_m max_i Cbar_mi via per-block partials
// reduced in order by the last block.
__global__ void __launch_bounds__(256) objective_kernel(Shape sh, Ws ws) {
  __shared__ float red[16];
  __shared__ int flag;
  const int p = blockIdx.y, m = blockIdx.x * 256 + threadIdx.x;
  float c = 0.f, pk = 0.f;
  if (m < sh.m) {
    c = ws.cov[p * ws.s_cov + m];
    pk = ws.peak[p * ws.s_m + m];
  }
  const float fs = block_sum(c, red);
  const float fv = block_sum(pk, red);
  float* sp = ws.spart + p * ws.s_spart;
  if (threadIdx.x == 0) {
    st_dev(&sp[2 * blockIdx.x], fs);
    st_dev(&sp[2 * blockIdx.x + 1], fv);
  }
  int* cnt = ws.cnt + p * ws.s_cnt;
  if (!last_arrival(&cnt[2], gridDim.x, &flag)) return;
  if (threadIdx.x == 0) {
    st_dev(&cnt[2], 0);
    float a = 0.f, b = 0.f;
#pragma unroll 8
    for (unsigned k = 0; k < gridDim.x; ++k) { a += ld_dev(&sp[2 * k]); b += ld_dev(&sp[2 * k + 1]); }
    float* st = ws.stats + p * ws.s_st;
    st[2] = a;
    st[3] = b;
    st[4] = static_cast<float>(sh.K);
    st[5] = static_cast<float>(sh.rounds);
    st[6] = static_cast<float>(sh.m);
    st[7] = static_cast<float>(sh.N - sh.K);
  }
}


static void launch_cov(const Shape& sh, const Ws& ws, int nb, hipStream_t st) {
  hipLaunchKernelGGL(cov_kernel, dim3((sh.m + 255) / 256, (nb + kCovCols - 1) / kCovCols, sh.B), dim3(256), 0,
                     st, sh, ws, nb);
}

// Blocks per problem for the persistent selection, or 0 when the call does
// not qualify (large pools, keys beyond LDS).  The grid never exceeds what
// the device holds at once (one block per CU, checked against the kernel's
// occupancy), so on a device not shared with other work every block is
// resident from the start.  The launch is an ordinary one: a cooperative
// launch costs a cross-queue synchronisation on each side of the kernel, and
// the bounded barrier waits already turn a block that never becomes resident
// (a device saturated by foreign work) into a reported timeout rather than a
// hang.
static const void* persistent_fn(int res) {
  return res ? reinterpret_cast<const void*>(select_persistent_kernel<true>)
             : reinterpret_cast<const void*>(select_persistent_kernel<false>);
}

static int g_n_cu = -1;   // compute units of the current device (0: unknown)

static int persistent_blocks(const Shape& sh, size_t lds, int res) {
  static int lds_max = 0, lds_set[2] = {64 * 1024, 64 * 1024};
  int& n_cu = g_n_cu;
  if (n_cu < 0) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
      n_cu = 0;
  }
  if (n_cu <= 0 || sh.pool_cap > 64 || sh.N > kLdsKeys || lds > static_cast<size_t>(lds_max)) return 0;
  const int v = res ? 1 : 0;
  if (static_cast<int>(lds) > lds_set[v]) {
    // dynamic LDS above 64 KB has to be granted to the kernel first
    if (hipFuncSetAttribute(persistent_fn(res), hipFuncAttributeMaxDynamicSharedMemorySize,
                            static_cast<int>(lds)) != hipSuccess)
      return 0;
    lds_set[v] = static_cast<int>(lds);
  }
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, persistent_fn(res), 256, lds) != hipSuccess || per_cu < 1)
    return 0;
  // about two gain tokens per wave; one block per CU, or two when the
  // streamed (non-resident) kernel fits twice, which doubles the waves that
  // stream the client rows
  const int cap = (res ? 1 : std::min(per_cu, 2)) * n_cu / sh.B;
  const int want = max((sh.N + 7) / 8, ((sh.m + 63) / 64 + 3) / 4);
  const int nblk = min(min(cap, want), kMaxPersist);
  return nblk >= 1 ? nblk : 0;
}

hipError_t launch_selection(const Shape& sh, const Params& pr, const Ws& ws, const SelOut& so, hipStream_t st,
                            bool* support_ready) {
  *support_ready = false;
  if (sh.rounds == 0) {
    // the image seeds already fill the budget (K = I): only the objective;
    // the assignment builds the support list from the selection marks
    timer_mark(kStObjective, true, st);
    hipLaunchKernelGGL(objective_kernel, dim3((sh.m + 255) / 256, sh.B), dim3(256), 0, st, sh, ws);
    timer_mark(kStObjective, false, st);
    return hipGetLastError();
  }
  {
    const size_t lds = static_cast<size_t>(sh.ldM) * sizeof(float) +
                       ((static_cast<size_t>(sh.N) + 15) & ~static_cast<size_t>(15)) +
                       (sh.N > 256 * 16 ? static_cast<size_t>(sh.N) * sizeof(uint32_t) : 0);
    int nblk = persistent_blocks(sh, lds, 0);
    // the blocks' client rows held in registers when each block owns at
    // most eight tokens and the rows are short enough
    const bool resident = nblk > 0 && sh.N <= 8 * nblk && sh.m <= 256 * kResJ &&
                          persistent_blocks(sh, lds, 1) == nblk;
    if (nblk > 0) {
      timer_mark(kStSelect, true, st);
      // the streamed gains take four tokens per wave pass when the grid has
      // one block per CU (registers to spare); with two per CU the two-token
      // loop measured faster
      const int quad = !resident && g_n_cu > 0 && nblk * sh.B <= g_n_cu;
      if (resident)
        hipLaunchKernelGGL(select_persistent_kernel<true>, dim3(nblk, sh.B), dim3(256), lds, st, sh, pr, ws,
                           nblk, so, 0);
      else
        hipLaunchKernelGGL(select_persistent_kernel<false>, dim3(nblk, sh.B), dim3(256), lds, st, sh, pr, ws, nblk,
                           so, quad);
      timer_mark(kStSelect, false, st);
      *support_ready = true;
      return hipGetLastError();
    }
  }
  const bool global_keys = sh.N > kLdsKeys;
  const size_t key_lds = global_keys ? 0 : static_cast<size_t>(sh.N) * sizeof(uint32_t);
  // unfused rounds pick the pool in a 1024-thread register top-k kernel
  // (keys per thread: 4, 8 or 16); beyond 16 * 1024 tokens the gains
  // kernel's last block does it over keys in global memory
  const int pool_seg = (sh.N + 64 * kPoolW - 1) / (64 * kPoolW);
  const int pool_kpt = pool_seg <= 4 ? 4 : pool_seg <= 8 ? 8 : pool_seg <= 16 ? 16 : 0;
  static int pool_lds_granted = 48 * 1024;
  const size_t fused_lds = static_cast<size_t>(sh.ldM) * sizeof(float) + key_lds;
  // small pools fuse the batch pick and the coverage refresh into the gains
  // kernel while the refreshed coverage fits in LDS next to the keys
  // fused only while the call is latency-bound: every fused block re-reads
  // the batch columns, which costs more than a launch once the client
  // matrix is large
  const long long cbar_bytes = 4LL * sh.B * sh.N * sh.m;
  const bool fused = sh.pool_cap <= 64 && fused_lds <= 56 * 1024 && cbar_bytes <= (48LL << 20);
  const dim3 gg((sh.N + kGainCols - 1) / kGainCols, sh.B);
  const dim3 ggf((sh.N + kGainColsF - 1) / kGainColsF, sh.B);
  int selected = sh.nseed, prev_psize = 0, prev_bsize = 0, prev_base = 0;
  for (int r = 0; r < sh.rounds; ++r) {
    const int psize = min(sh.pool_cap, sh.N - selected);
    const int bsize = min(sh.b, sh.K - selected);
    if (fused) {
      timer_mark(kStGains, true, st);
      if (global_keys)
        hipLaunchKernelGGL(gains_fused_kernel<true>, ggf, dim3(256), fused_lds, st, sh, ws, r, psize,
                           prev_psize, prev_bsize, prev_base, so);
      else
        hipLaunchKernelGGL(gains_fused_kernel<false>, ggf, dim3(256), fused_lds, st, sh, ws, r, psize,
                           prev_psize, prev_bsize, prev_base, so);
      timer_mark(kStGains, false, st);
      timer_mark(kStResp, true, st);
      hipLaunchKernelGGL(resp_small_kernel, dim3((sh.m + 255) / 256, sh.B), dim3(256), 0, st, sh, pr, ws,
                         psize);
      timer_mark(kStResp, false, st);
    } else {
      if (r > 0) {
        timer_mark(kStCov, true, st);
        launch_cov(sh, ws, sh.b, st);
        timer_mark(kStCov, false, st);
      }
      timer_mark(kStGains, true, st);
      if (pool_kpt > 0) {
        hipLaunchKernelGGL((gains_kernel<true, false>), gg, dim3(256), 0, st, sh, ws, r, psize, so);
        // the pool's own kernel is timed with the responsibilities
        timer_mark(kStGains, false, st);
        timer_mark(kStResp, true, st);
        const dim3 gp(sh.B), bp(64 * kPoolW);
        const size_t pl = static_cast<size_t>(sh.N) * sizeof(uint32_t);
        if (pool_kpt == 16 && static_cast<int>(pl) > pool_lds_granted) {
          // 64 KB of keys next to the static histograms: grant the dynamic LDS once
          const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(pool_topk_kernel<16>),
                                                   hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(pl));
          if (e != hipSuccess) return e;
          pool_lds_granted = static_cast<int>(pl);
        }
        if (pool_kpt == 4)
          hipLaunchKernelGGL(pool_topk_kernel<4>, gp, bp, pl, st, sh, ws, r, psize, so);
        else if (pool_kpt == 8)
          hipLaunchKernelGGL(pool_topk_kernel<8>, gp, bp, pl, st, sh, ws, r, psize, so);
        else
          hipLaunchKernelGGL(pool_topk_kernel<16>, gp, bp, pl, st, sh, ws, r, psize, so);
      } else {
        if (global_keys)
          hipLaunchKernelGGL(gains_kernel<true>, gg, dim3(256), 0, st, sh, ws, r, psize, so);
        else
          hipLaunchKernelGGL(gains_kernel<false>, gg, dim3(256), key_lds, st, sh, ws, r, psize, so);
        timer_mark(kStGains, false, st);
        timer_mark(kStResp, true, st);
      }
      if (sh.pool_cap <= 64)
        hipLaunchKernelGGL(resp_small_kernel, dim3((sh.m + 255) / 256, sh.B), dim3(256), 0, st, sh, pr, ws,
                           psize);
      else {
        hipLaunchKernelGGL(rowstat_kernel, dim3((sh.m + 63) / 64, sh.B), dim3(64 * kRsW), 0, st, sh, pr, ws, psize);
        hipLaunchKernelGGL(colsum_kernel, dim3((psize + 3) / 4, sh.B), dim3(256),
                           static_cast<size_t>(sh.pool_cap) * sizeof(uint32_t), st, sh, ws, r, psize, bsize,
                           selected, so);
      }
      if (sh.pool_cap <= 64)
        hipLaunchKernelGGL(final_batch_kernel, dim3(sh.B), dim3(64), 0, st, sh, ws, r, psize, bsize, selected,
                           so);
      timer_mark(kStResp, false, st);
    }
    prev_psize = psize;
    prev_bsize = bsize;
    prev_base = selected;
    selected += bsize;
  }
  timer_mark(kStObjective, true, st);
  if (fused)
    hipLaunchKernelGGL(final_batch_kernel, dim3(sh.B), dim3(64), 0, st, sh, ws, sh.rounds - 1, prev_psize,
                       prev_bsize, prev_base, so);
  launch_cov(sh, ws, prev_bsize, st);
  hipLaunchKernelGGL(objective_kernel, dim3((sh.m + 255) / 256, sh.B), dim3(256), 0, st, sh, ws);
  timer_mark(kStObjective, false, st);
  return hipGetLastError();
}

}  // namespace gmc
