// Device-side helpers shared by the GMC kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gmc {

typedef uint16_t bf16_t;  // bfloat16 stored as its bit pattern
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf16_to_f32(bf16_t v) {
  return __uint_as_float(static_cast<uint32_t>(v) << 16);
}

// Round-to-nearest-even float -> bf16 (finite inputs).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<bf16_t>(u >> 16);
}

template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<bf16_t>(bf16_t v) { return bf16_to_f32(v); }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) { return f32_to_bf16(v); }

// ---------------------------------------------------------------------------
// wave64 scans and reductions on DPP row operations (gfx9 family):
// row_shr:n moves values n lanes up inside each 16-lane row, row_bcast:15
// and row_bcast:31 carry a row's last lane into the following rows.  Lanes
// without a source keep `old` (the operation's identity).  A reduction is the
// inclusive scan's last lane, read back as a wave-uniform value.
// ---------------------------------------------------------------------------
template <int kCtrl, int kRowMask>
__device__ __forceinline__ int dpp_i(int old, int v) {
  return __builtin_amdgcn_update_dpp(old, v, kCtrl, kRowMask, 0xf, false);
}
template <int kCtrl, int kRowMask>
__device__ __forceinline__ float dpp_f(float old, float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(v), kCtrl, kRowMask, 0xf,
                                                    false));
}
#define GMC_WAVE_SCAN(T, DPP, ID, OP)          \
  v = OP(v, DPP<0x111, 0xf>(ID, v));           \
  v = OP(v, DPP<0x112, 0xf>(ID, v));           \
  v = OP(v, DPP<0x114, 0xf>(ID, v));           \
  v = OP(v, DPP<0x118, 0xf>(ID, v));           \
  v = OP(v, DPP<0x142, 0xa>(ID, v));           \
  v = OP(v, DPP<0x143, 0xc>(ID, v));           \
  return v;

__device__ __forceinline__ int op_add_i(int a, int b) { return a + b; }
__device__ __forceinline__ float op_add_f(float a, float b) { return a + b; }
__device__ __forceinline__ int op_and_i(int a, int b) { return a & b; }
__device__ __forceinline__ int op_or_i(int a, int b) { return a | b; }

// Inclusive prefix sums over the 64 lanes.
__device__ __forceinline__ int wave_scan_add(int v) { GMC_WAVE_SCAN(int, dpp_i, 0, op_add_i) }
__device__ __forceinline__ float wave_scan_addf(float v) { GMC_WAVE_SCAN(float, dpp_f, 0.f, op_add_f) }
__device__ __forceinline__ float wave_scan_maxf(float v) { GMC_WAVE_SCAN(float, dpp_f, -INFINITY, fmaxf) }
__device__ __forceinline__ float wave_scan_minf(float v) { GMC_WAVE_SCAN(float, dpp_f, INFINITY, fminf) }
__device__ __forceinline__ int wave_scan_and(int v) { GMC_WAVE_SCAN(int, dpp_i, -1, op_and_i) }
__device__ __forceinline__ int wave_scan_or(int v) { GMC_WAVE_SCAN(int, dpp_i, 0, op_or_i) }
#undef GMC_WAVE_SCAN

// The wave's index in its block as a wave-uniform (scalar) value, so that
// tile indices derived from it branch and address in scalar registers.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6)); }

__device__ __forceinline__ float lane63(float v) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}
__device__ __forceinline__ float wave_sum(float v) { return lane63(wave_scan_addf(v)); }
__device__ __forceinline__ float wave_max(float v) { return lane63(wave_scan_maxf(v)); }
__device__ __forceinline__ float wave_min(float v) { return lane63(wave_scan_minf(v)); }
__device__ __forceinline__ int wave_sum_i(int v) { return __builtin_amdgcn_readlane(wave_scan_add(v), 63); }
__device__ __forceinline__ uint32_t wave_and_u(uint32_t v) {
  return static_cast<uint32_t>(__builtin_amdgcn_readlane(wave_scan_and(static_cast<int>(v)), 63));
}
__device__ __forceinline__ uint32_t wave_or_u(uint32_t v) {
  return static_cast<uint32_t>(__builtin_amdgcn_readlane(wave_scan_or(static_cast<int>(v)), 63));
}
// The value of lane l ^ O (O < 16) by DPP moves, no LDS round trip: quad
// permutations for 1 and 2; 4 and 8 compose a quad reversal (l ^ 3) or a row
// mirror (l ^ 15) with a half-row mirror (l ^ 7).
template <int O>
__device__ __forceinline__ float xor_lane(float v) {
  static_assert(O == 1 || O == 2 || O == 4 || O == 8 || O == 16 || O == 32, "lane exchange by a power of two");
  if constexpr (O == 1) return dpp_f<0xB1, 0xf>(v, v);
  if constexpr (O == 2) return dpp_f<0x4E, 0xf>(v, v);
  if constexpr (O == 4) return dpp_f<0x141, 0xf>(v, dpp_f<0x1B, 0xf>(v, v));
  if constexpr (O == 8) return dpp_f<0x141, 0xf>(v, dpp_f<0x140, 0xf>(v, v));
  // 16 and 32: a permlane swap of two copies leaves the lane's own value in
  // one result and its partner's in the other, by the lane's half
  if constexpr (O == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(((threadIdx.x >> 4) & 1) ? r[0] : r[1]);
  }
  if constexpr (O == 32) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(((threadIdx.x >> 5) & 1) ? r[0] : r[1]);
  }
  return v;
}
template <int O>
__device__ __forceinline__ int xor_lane_i(int v) {
  return __float_as_int(xor_lane<O>(__int_as_float(v)));
}

// v[l] + v[l ^ 16] and v[l] + v[l ^ 32] in every lane: a permlane swap of two
// copies of v puts the partner's value beside the lane's own (the order of
// the two terms differs between halves; the sum does not).
__device__ __forceinline__ float add_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float add_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Reduce across the 16 lanes of one MFMA row group (lanes l with equal l/16)
// with DPP moves: two quad butterflies, then rotations by 4 and 8 inside the
// 16-lane row.  Every lane receives the reduction; for sums the association
// differs between the row's quads, so callers take one fixed lane's value.
__device__ __forceinline__ float group16_sum(float v) {
  v += dpp_f<0xB1, 0xf>(0.f, v);    // quad_perm [1, 0, 3, 2]
  v += dpp_f<0x4E, 0xf>(0.f, v);    // quad_perm [2, 3, 0, 1]
  v += dpp_f<0x124, 0xf>(0.f, v);   // row_ror:4
  v += dpp_f<0x128, 0xf>(0.f, v);   // row_ror:8
  return v;
}
__device__ __forceinline__ float group16_max(float v) {
  v = fmaxf(v, dpp_f<0xB1, 0xf>(v, v));
  v = fmaxf(v, dpp_f<0x4E, 0xf>(v, v));
  v = fmaxf(v, dpp_f<0x124, 0xf>(v, v));
  v = fmaxf(v, dpp_f<0x128, 0xf>(v, v));
  return v;
}

// Sum over a whole block (blockDim.x multiple of 64, <= 1024). `red` holds
// >= 16 floats of LDS.  Deterministic: fixed shuffle tree, then waves in order.
__device__ __forceinline__ float block_sum(float v, float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
  for (int i = 0; i < nw; ++i) s += red[i];
  return s;
}
__device__ __forceinline__ float block_max(float v, float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_max(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float s = -INFINITY;
  for (int i = 0; i < nw; ++i) s = fmaxf(s, red[i]);
  return s;
}
__device__ __forceinline__ float block_min(float v, float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_min(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float s = INFINITY;
  for (int i = 0; i < nw; ++i) s = fminf(s, red[i]);
  return s;
}

// Exclusive prefix sum of one int per thread over the block; returns the
// exclusive prefix and writes the block total to *total.  `scan` holds >= 16
// ints of LDS.
__device__ __forceinline__ int block_exclusive_scan(int v, int* scan, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int incl = wave_scan_add(v);
  __syncthreads();
  if (lane == 63) scan[w] = incl;
  __syncthreads();
  int base = 0, tot = 0;
  for (int i = 0; i < nw; ++i) {
    if (i < w) base += scan[i];
    tot += scan[i];
  }
  *total = tot;
  return base + incl - v;
}

// ---------------------------------------------------------------------------
// MFMA 16x16x32 step with a uniform operand layout for bf16 and fp32.
// Lane l supplies 8 consecutive k-elements (k-block l/16) of row (A) or
// column (B) l%16.  The output 16x16 tile: lane l holds column l%16, rows
// 4*(l/16) + 0..3.  For fp32 the step is eight 16x16x4 MFMAs; the k-slot
// assignment is the same for A and B, so every product appears once.
// ---------------------------------------------------------------------------
template <typename T> struct Frag;
template <> struct Frag<bf16_t> { bf16x8 v; };
template <> struct Frag<float> { float v[8]; };

template <typename T> __device__ __forceinline__ Frag<T> frag_load(const T* p);
template <> __device__ __forceinline__ Frag<bf16_t> frag_load<bf16_t>(const bf16_t* p) {
  Frag<bf16_t> f;
  f.v = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
  return f;
}
template <> __device__ __forceinline__ Frag<float> frag_load<float>(const float* p) {
  Frag<float> f;
  const float4 a = reinterpret_cast<const float4*>(p)[0];
  const float4 b = reinterpret_cast<const float4*>(p)[1];
  f.v[0] = a.x; f.v[1] = a.y; f.v[2] = a.z; f.v[3] = a.w;
  f.v[4] = b.x; f.v[5] = b.y; f.v[6] = b.z; f.v[7] = b.w;
  return f;
}
template <typename T> __device__ __forceinline__ Frag<T> frag_zero();
template <> __device__ __forceinline__ Frag<bf16_t> frag_zero<bf16_t>() {
  Frag<bf16_t> f;
  f.v = __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0));
  return f;
}
template <> __device__ __forceinline__ Frag<float> frag_zero<float>() {
  Frag<float> f;
#pragma unroll
  for (int j = 0; j < 8; ++j) f.v[j] = 0.f;
  return f;
}

__device__ __forceinline__ floatx4 mma(const Frag<bf16_t>& a, const Frag<bf16_t>& b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, c, 0, 0, 0);
}
__device__ __forceinline__ floatx4 mma(const Frag<float>& a, const Frag<float>& b, floatx4 c) {
#pragma unroll
  for (int j = 0; j < 8; ++j) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[j], b.v[j], c, 0, 0, 0);
  return c;
}

// 16-byte global<->LDS chunk copies (8 bf16 or 4 floats).
__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }
__device__ __forceinline__ void st16(void* p, uint4 v) { *reinterpret_cast<uint4*>(p) = v; }
// Eight consecutive elements (16-byte aligned) as fp32, and back.
template <typename T> __device__ __forceinline__ void load8_f32(const T* p, float* v);
template <> __device__ __forceinline__ void load8_f32<bf16_t>(const bf16_t* p, float* v) {
  const uint4 raw = ld16(p);
  const bf16_t* b = reinterpret_cast<const bf16_t*>(&raw);
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = bf16_to_f32(b[e]);
}
template <> __device__ __forceinline__ void load8_f32<float>(const float* p, float* v) {
  const uint4 r0 = ld16(p), r1 = ld16(p + 4);
  const float* a = reinterpret_cast<const float*>(&r0);
  const float* b = reinterpret_cast<const float*>(&r1);
#pragma unroll
  for (int e = 0; e < 4; ++e) { v[e] = a[e]; v[e + 4] = b[e]; }
}
template <typename T> __device__ __forceinline__ void store8_f32(T* p, const float* v);
template <> __device__ __forceinline__ void store8_f32<bf16_t>(bf16_t* p, const float* v) {
  uint4 raw;
  bf16_t* b = reinterpret_cast<bf16_t*>(&raw);
#pragma unroll
  for (int e = 0; e < 8; ++e) b[e] = f32_to_bf16(v[e]);
  st16(p, raw);
}
template <> __device__ __forceinline__ void store8_f32<float>(float* p, const float* v) {
  st16(p, make_uint4(__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]), __float_as_uint(v[3])));
  st16(p + 4, make_uint4(__float_as_uint(v[4]), __float_as_uint(v[5]), __float_as_uint(v[6]), __float_as_uint(v[7])));
}

// Device-coherent hand-off between blocks of one kernel.  Data another block
// reads in the same launch is written with agent-scope relaxed atomic stores
// (write-through past the per-XCD L2) and read with agent-scope atomic loads,
// so no L2 writeback/invalidate is needed; ordering against the completion
// counter comes from waiting for this wave's stores before the block barrier.
__device__ __forceinline__ void st_dev(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_dev(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void st_dev64(unsigned long long* p, unsigned long long v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long ld_dev64(const unsigned long long* p) {
  return __hip_atomic_load(const_cast<unsigned long long*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// A float with a 32-bit tag in the high word (one 8-byte atomic access).
__device__ __forceinline__ unsigned long long tag_value(unsigned tag, float v) {
  return (static_cast<unsigned long long>(tag) << 32) | __float_as_uint(v);
}
__device__ __forceinline__ unsigned tag_of(unsigned long long w) { return static_cast<unsigned>(w >> 32); }
__device__ __forceinline__ float value_of(unsigned long long w) {
  return __uint_as_float(static_cast<unsigned>(w & 0xFFFFFFFFull));
}

// Last-block detection: every wave waits until its device-coherent stores
// have completed, then one counter increment per block; returns true in the
// block that completes `total` arrivals (uniform across the block).
__device__ __forceinline__ bool last_arrival(int* counter, int total, int* flag) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0)
    *flag = (__hip_atomic_fetch_add(counter, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == total - 1) ? 1 : 0;
  __syncthreads();
  return *flag != 0;
}

// Four floats from a 16-byte aligned address with a non-temporal (streaming)
// load: data read once that should not displace cached lines.
__device__ __forceinline__ float4 ld_stream4(const float* ptr) {
  typedef float f32x4_t __attribute__((ext_vector_type(4)));
  const f32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(ptr));
  return make_float4(v.x, v.y, v.z, v.w);
}

// Order-preserving key of a non-negative float score (larger score -> larger
// key); 0 is reserved for excluded candidates.
__device__ __forceinline__ uint32_t score_key(float s) { return __float_as_uint(fmaxf(s, 0.f)) + 1u; }

}  // namespace gmc
