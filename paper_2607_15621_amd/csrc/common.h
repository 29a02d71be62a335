// Device-side building blocks shared by the kernels of the expert tick (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/fsx.h"

namespace fsx {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8;
typedef __attribute__((__vector_size__(2 * sizeof(_Float16)))) _Float16 f16x2;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

constexpr int WAVE = 64;
constexpr float LOG2E = 1.4426950408889634f;

// ---------------------------------------------------------------- scalar conversions

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2_t;

// round-to-nearest-even float -> bf16 bits (NaN stays NaN): one v_cvt_pk_bf16_f32 on gfx950
__device__ __forceinline__ uint16_t f32_to_bf16(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

// two floats -> packed bf16x2 (RNE), low half = a
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const bf16x2_t v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ uint32_t pack_f16x2(float a, float b) {
  _Float16 ha = (_Float16)a, hb = (_Float16)b;
  return (uint32_t)__builtin_bit_cast(uint16_t, ha) | ((uint32_t)__builtin_bit_cast(uint16_t, hb) << 16);
}

// OCP E4M3 (e4m3fn) pair -> f16x2, exact (every E4M3 value is an fp16 value).  `word` selects
// bytes 0-1 (false) or 2-3 (true) of `packed`.
__device__ __forceinline__ uint32_t e4m3x2_to_f16x2(uint32_t packed, bool word) {
  f16x2 r = word ? __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(packed, 1.0f, true)
                 : __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(packed, 1.0f, false);
  return __builtin_bit_cast(uint32_t, r);
}

__device__ __forceinline__ float e4m3_to_f32(uint8_t c) {
  uint32_t p = c;
  f16x2 r = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(p, 1.0f, false);
  return (float)r[0];
}

// ---------------------------------------------------------------- MFMA (16x16x32, fp32 accumulate)
// Operand layout (wave64): lane l holds A[row = l%16][k = 8*(l/16) + j] and
// B[k = 8*(l/16) + j][col = l%16], j = 0..7; the result lane l holds
// C[row = 4*(l/16) + i][col = l%16], i = 0..3.

__device__ __forceinline__ f32x4 mfma_bf16(uint4 a, uint4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                 0, 0, 0);
}

__device__ __forceinline__ f32x4 mfma_f16(uint4 a, uint4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                0, 0);
}

// ---------------------------------------------------------------- cross-lane helpers
// No cross-lane move in these kernels goes through the LDS crossbar (ds_bpermute, ds_swizzle: what __shfl and
// __shfl_xor compile to).  In a wave whose direct loads into LDS were still landing, such shuffles returned wrong
// values now and then (the attention's running-max rescale gave launch-to-launch differences); DPP, the permlane
// swaps and readlane do not use the LDS path.

// Cross-lane moves without the LDS crossbar (DPP and the gfx950 permlane swaps):
//   xor1(v)      value of lane l ^ 1 (quad_perm [1,0,3,2])
//   xor8(v)      value of lane l ^ 8 (row_ror:8 inside each 16-lane row)
//   row_sum16(v) sum over the 16 lanes of l's row, in every lane (rotations by 8, 4, 2, 1)
//   rows_max/rows_sum(v): max / sum over lanes l, l ^ 16, l ^ 32, l ^ 48 (permlane16_swap then permlane32_swap;
//   each swap of v with itself returns the two halves of the exchange, combined by the operation)
__device__ __forceinline__ float xor1(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false));
}
__device__ __forceinline__ float xor8(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x128, 0xF, 0xF, false));
}
__device__ __forceinline__ float row_sum16(float v) {
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x128, 0xF, 0xF, false));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x124, 0xF, 0xF, false));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x122, 0xF, 0xF, false));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x121, 0xF, 0xF, false));
  return v;
}
// Maximum by the hardware instruction alone, without the quieting of signalling NaNs that fmaxf adds (the attention
// scores it is used on are never NaN unless the inputs are).
__device__ __forceinline__ float vmax(float a, float b) {
  float r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ __forceinline__ float vmax3(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}
__device__ __forceinline__ float rows_max(float v) {
  const unsigned u = __builtin_bit_cast(unsigned, v);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const float m = vmax(__builtin_bit_cast(float, (unsigned)a[0]), __builtin_bit_cast(float, (unsigned)a[1]));
  const unsigned mu = __builtin_bit_cast(unsigned, m);
  const auto b = __builtin_amdgcn_permlane32_swap(mu, mu, false, false);
  return vmax(__builtin_bit_cast(float, (unsigned)b[0]), __builtin_bit_cast(float, (unsigned)b[1]));
}
__device__ __forceinline__ float rows_sum(float v) {
  const unsigned u = __builtin_bit_cast(unsigned, v);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const float m = __builtin_bit_cast(float, (unsigned)a[0]) + __builtin_bit_cast(float, (unsigned)a[1]);
  const unsigned mu = __builtin_bit_cast(unsigned, m);
  const auto b = __builtin_amdgcn_permlane32_swap(mu, mu, false, false);
  return __builtin_bit_cast(float, (unsigned)b[0]) + __builtin_bit_cast(float, (unsigned)b[1]);
}
// Sum over the 64 lanes, in every lane.
__device__ __forceinline__ float wave_sum(float v) { return rows_sum(row_sum16(v)); }
// For the lanes of 16-lane row grp: the value of lane 4 grp + i, where lanes 0..15 hold one value per column and
// every row repeats them (a per-query running statistic); four lane reads selected by row.
__device__ __forceinline__ float col_pick(float v, int grp, int i) {
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), i));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 4 + i));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 8 + i));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 12 + i));
  return grp == 0 ? r0 : (grp == 1 ? r1 : (grp == 2 ? r2 : r3));
}

// Transpose an 8x8 block of 16-bit values held as 8 x uint4 (in[j] = row j, 8 columns) into
// out[k] = column k as 8 values (element j = in[j][k]).
__device__ __forceinline__ void transpose8x8_b16(const uint4 in[8], uint4 out[8]) {
  const uint32_t* w = reinterpret_cast<const uint32_t*>(in);  // w[j*4 + k/2]
  uint32_t* o = reinterpret_cast<uint32_t*>(out);            // o[k*4 + j/2]
#pragma unroll
  for (int k = 0; k < 8; ++k) {
#pragma unroll
    for (int jp = 0; jp < 4; ++jp) {
      uint32_t lo = w[(2 * jp) * 4 + k / 2];
      uint32_t hi = w[(2 * jp + 1) * 4 + k / 2];
      o[k * 4 + jp] = __builtin_amdgcn_perm(hi, lo, (k & 1) ? 0x07060302u : 0x05040100u);
    }
  }
}

// ---------------------------------------------------------------- device-coherent accesses
// Data exchanged between workgroups inside one launch is written with device-scope ("sc1") stores,
// which write through the XCD's L2 to memory, and read with device-scope loads, which do not return
// lines cached by another XCD's L2.  A producer waits for its stores to complete (stores_done) before
// it publishes a flag; no L2 write-back or invalidate is needed.
__device__ __forceinline__ void st_dev(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev_f(float* p, float v) { st_dev(reinterpret_cast<uint32_t*>(p), __float_as_uint(v)); }
__device__ __forceinline__ void st_dev16(void* p, uint4 v) {
  uint64_t* q = reinterpret_cast<uint64_t*>(p);
  st_dev(q, (uint64_t)v.x | ((uint64_t)v.y << 32));
  st_dev(q + 1, (uint64_t)v.z | ((uint64_t)v.w << 32));
}
__device__ __forceinline__ void st_dev_f4(float* p, float4 v) {
  st_dev16(p, make_uint4(__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z), __float_as_uint(v.w)));
}
__device__ __forceinline__ uint32_t ld_dev(const uint32_t* p) {
  return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_dev(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_dev_f(const float* p) { return __uint_as_float(ld_dev(reinterpret_cast<const uint32_t*>(p))); }
__device__ __forceinline__ uint4 ld_dev16(const void* p) {
  const uint64_t* q = reinterpret_cast<const uint64_t*>(p);
  const uint64_t a = ld_dev(q), b = ld_dev(q + 1);
  return make_uint4((uint32_t)a, (uint32_t)(a >> 32), (uint32_t)b, (uint32_t)(b >> 32));
}
__device__ __forceinline__ float4 ld_dev_f4(const float* p) {
  const uint4 u = ld_dev16(p);
  return make_float4(__uint_as_float(u.x), __uint_as_float(u.y), __uint_as_float(u.z), __uint_as_float(u.w));
}
// Wait until every vector memory operation this thread issued has completed (s_waitcnt vmcnt(0), GFX9
// encoding).  Through the builtin, so the compiler knows those loads are complete and adds no later wait
// for them; the empty asm statements keep memory accesses from moving across it.
__device__ __forceinline__ void vm_wait_all() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0x0F70);
  asm volatile("" ::: "memory");
}
__device__ __forceinline__ void stores_done() { vm_wait_all(); }
// Wait until at most N (< 64) of this thread's vector memory operations are pending: they complete in issue order,
// so everything issued before the last N has completed.
template <int N>
__device__ __forceinline__ void vm_wait_below_c() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
  asm volatile("" ::: "memory");
}

// Stores of data exchanged between workgroups of ONE XCD: plain stores, which stay in the XCD's L2 (the
// vector L1 is write-through); readers use device-scope loads, which are served by that L2 and never by a
// stale L1 line.  A producer waits for the stores (stores_done) before it publishes a flag.
__device__ __forceinline__ void st_loc(uint32_t* p, uint32_t v) { *p = v; }
__device__ __forceinline__ void st_loc(uint64_t* p, uint64_t v) { *p = v; }
__device__ __forceinline__ void st_loc_f(float* p, float v) { st_loc(reinterpret_cast<uint32_t*>(p), __float_as_uint(v)); }
__device__ __forceinline__ void st_loc16(void* p, uint4 v) { *reinterpret_cast<uint4*>(p) = v; }
__device__ __forceinline__ void st_loc_f4(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }

// Load through a pointer that addresses global memory.  A pointer the compiler cannot prove global (one
// read from memory, such as a table of weight pointers) would otherwise give a flat load, which also counts
// in the LDS counter, so every later LDS wait would wait for it too.
// (Through a native vector type: a cast of a pointer to the class type uint4 loses its address space.)
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld_global(const uint4* p) {
  const u32x4_t v = *(const __attribute__((address_space(1))) u32x4_t*)p;
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Direct load global -> LDS of 16 bytes per lane: lane l's 16 bytes at src land at lds_base + 16 l
// (lds_base is wave-uniform).  No registers hold the data; completion is counted by vmcnt.
// COH: device-scope (sc1) load, for data produced inside the same launch.
template <bool COH = false>
__device__ __forceinline__ void load_lds16(const void* src, void* lds_base) {
  typedef __attribute__((address_space(3))) void lds_void_t;
  typedef const __attribute__((address_space(1))) void g_void_t;
  __builtin_amdgcn_global_load_lds((g_void_t*)src, (lds_void_t*)lds_base, 16, 0, COH ? 16 : 0);
}

// Plain or device-coherent access, chosen at compile time.
template <bool COH>
__device__ __forceinline__ uint4 ld16(const void* p) {
  if constexpr (COH) return ld_dev16(p);
  else return *reinterpret_cast<const uint4*>(p);
}
template <bool COH>
__device__ __forceinline__ float4 ldf4(const float* p) {
  if constexpr (COH) return ld_dev_f4(p);
  else return *reinterpret_cast<const float4*>(p);
}
template <bool COH>
__device__ __forceinline__ float ldf(const float* p) {
  if constexpr (COH) return ld_dev_f(p);
  else return *p;
}
template <bool COH>
__device__ __forceinline__ void stf(float* p, float v) {
  if constexpr (COH) st_dev_f(p, v);
  else *p = v;
}
template <bool COH>
__device__ __forceinline__ void stf4(float* p, float4 v) {
  if constexpr (COH) st_dev_f4(p, v);
  else *reinterpret_cast<float4*>(p) = v;
}
template <bool COH>
__device__ __forceinline__ void st16(void* p, uint4 v) {
  if constexpr (COH) st_dev16(p, v);
  else *reinterpret_cast<uint4*>(p) = v;
}

__device__ __forceinline__ float block_sum(float v, float* scratch /* >= 16 floats */) {
  v = wave_sum(v);
  const int wave = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
  const int nw = (blockDim.x + WAVE - 1) / WAVE;
  __syncthreads();
  if (lane == 0) scratch[wave] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += scratch[i];
  return t;
}

}  // namespace fsx
