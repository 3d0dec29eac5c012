// Shared device helpers for the verify-step kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace nj {

typedef uint16_t bf16_t;  // bf16 storage (bit pattern)

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Split-K partials are exchanged between workgroups that may sit on different
// XCDs (separate L2s).  They are written and read as 16-byte buffer accesses
// with the device-coherence cache policy (sc1, the policy of agent-scope
// atomics), so no L2 writeback or invalidate is needed for the hand-off.
// Accesses past num_bytes are dropped (stores) or read as zero (loads).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t coherent_rsrc(void* base, int num_bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(base, (short)0, num_bytes, 0x00020000);
}
__device__ __forceinline__ void coherent_store(__amdgpu_buffer_rsrc_t r, uint32_t byte_off, f32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, byte_off, 0, 16 /* sc1 */);
}
__device__ __forceinline__ f32x4 coherent_load(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 16 /* sc1 */));
}

// Split-K partials inside one XCD (accelerator die: its CUs share one L2):
// a plain store reaches that L2, and an sc0 load skips the CU's L1 but may
// hit the L2, so workgroups on the same XCD exchange partials without a trip
// to memory.  Only valid between workgroups that are on the same XCD, which
// xcd_id() tells.
__device__ __forceinline__ void xcd_store(__amdgpu_buffer_rsrc_t r, uint32_t byte_off, f32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, byte_off, 0, 0);
}
__device__ __forceinline__ f32x4 xcd_load(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 1 /* sc0 */));
}
__device__ __forceinline__ unsigned xcd_id() {
  unsigned x;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
  return x & 0xfu;
}

__device__ __forceinline__ void coherent_store_f32(__amdgpu_buffer_rsrc_t r, uint32_t byte_off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), r, byte_off, 0, 16 /* sc1 */);
}
__device__ __forceinline__ float coherent_load_f32(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, byte_off, 0, 16 /* sc1 */));
}
__device__ __forceinline__ void coherent_store_f64(__amdgpu_buffer_rsrc_t r, uint32_t byte_off, double v) {
  __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, v), r, byte_off, 0, 16 /* sc1 */);
}
__device__ __forceinline__ double coherent_load_f64(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(double, __builtin_amdgcn_raw_buffer_load_b64(r, byte_off, 0, 16 /* sc1 */));
}

constexpr int kWave = 64;

// Softmax statistics of one 128-wide vocabulary chunk, computed by 8
// consecutive lanes holding 16 consecutive entries each (lane c of the group:
// entries 16c .. 16c+15; -inf marks entries past the vocabulary).  Every lane
// of the group returns the chunk max and the sum of exp(v - max), each formed
// in a fixed order, so the LM-head GEMM epilogue and the stand-alone
// statistics kernel produce the same bits.
constexpr int kStatChunk = 128, kStatLanes = 8, kStatPer = 16;
__device__ __forceinline__ void chunk_stats(const float (&v)[kStatPer], float& m, float& s) {
  m = v[0];
#pragma unroll
  for (int e = 1; e < kStatPer; ++e) m = fmaxf(m, v[e]);
  m = fmaxf(m, __shfl_xor(m, 1));
  m = fmaxf(m, __shfl_xor(m, 2));
  m = fmaxf(m, __shfl_xor(m, 4));
  s = 0.f;
#pragma unroll
  for (int e = 0; e < kStatPer; ++e) s += (v[e] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f((v[e] - m) * 1.4426950408889634f);
  s += __shfl_xor(s, 1);
  s += __shfl_xor(s, 2);
  s += __shfl_xor(s, 4);
}
constexpr int kBlock = 16;  // tokens per KV block

// Device error bits (mirror NJ_DEV_* of the public header).
constexpr int kErrToken = 1, kErrBlock = 2, kErrContext = 4, kErrAccept = 8, kErrSplitWait = 16;

__device__ __forceinline__ float bf2f(bf16_t v) { return __uint_as_float((uint32_t)v << 16); }

// fp32 -> bf16, round to nearest even (gfx950's v_cvt_pk_bf16_f32); NaN stays NaN.
__device__ __forceinline__ bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

__device__ __forceinline__ float to_f(float x) { return x; }
__device__ __forceinline__ float to_f(bf16_t x) { return bf2f(x); }

template <typename T> __device__ __forceinline__ T from_f(float x);
template <> __device__ __forceinline__ float from_f<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16_t from_f<bf16_t>(float x) { return f2bf(x); }

// Pack two fp32 into two bf16 in one dword (low = a), rounded to nearest
// even by one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ void flag_error(int* err, int bit) { atomicOr(err, bit); }

// Block-wide reductions (fixed order, so results are reproducible).
template <int NT>
__device__ __forceinline__ float block_sum(float v, float* sh) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int w = threadIdx.x / kWave, l = threadIdx.x % kWave;
  __syncthreads();
  if (l == 0) sh[w] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < NT / kWave; ++i) t += sh[i];
  return t;
}

template <int NT>
__device__ __forceinline__ float block_max(float v, float* sh) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  const int w = threadIdx.x / kWave, l = threadIdx.x % kWave;
  __syncthreads();
  if (l == 0) sh[w] = v;
  __syncthreads();
  float t = -INFINITY;
#pragma unroll
  for (int i = 0; i < NT / kWave; ++i) t = fmaxf(t, sh[i]);
  return t;
}

__device__ __forceinline__ double wave_sum_d(double v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

}  // namespace nj
