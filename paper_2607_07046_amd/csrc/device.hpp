// Device helpers for gfx950 (CDNA4): fp16 packing, wave/block reductions,
// agent-scope synchronisation words.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vt {

constexpr int kWave = 64;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float h2f(uint16_t u) {
  return static_cast<float>(__builtin_bit_cast(_Float16, u));
}

__device__ __forceinline__ uint16_t f2h(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<_Float16>(f));
}

// fp16 rounding of an fp32 value, returned as fp32.
__device__ __forceinline__ float round_h(float f) {
  return static_cast<float>(static_cast<_Float16>(f));
}

// The two fp16 numbers packed in a 32-bit word, as floats (low half first).
__device__ __forceinline__ void unpack2(unsigned w, float& a, float& b) {
  f16x2 h = __builtin_bit_cast(f16x2, w);
  a = static_cast<float>(h.x);
  b = static_cast<float>(h.y);
}

__device__ __forceinline__ void unpack8(const u32x4 v, float (&o)[8]) {
  unpack2(v.x, o[0], o[1]);
  unpack2(v.y, o[2], o[3]);
  unpack2(v.z, o[4], o[5]);
  unpack2(v.w, o[6], o[7]);
}

// Streaming 16-byte load of weights that are read exactly once per step.
__device__ __forceinline__ u32x4 load_stream(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

__device__ __forceinline__ u32x4 load16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// Sum over groups of ``width`` consecutive lanes (width a power of two <= 64).
__device__ __forceinline__ float group_sum(float v, int width) {
  for (int o = width >> 1; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// Block-wide sum in a fixed order; ``red`` is LDS of at least nwaves floats.
template <int NT>
__device__ __forceinline__ float block_sum(float v, float* red) {
  constexpr int NW = NT / kWave;
  v = wave_sum(v);
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NW; ++i) s += red[i];
  __syncthreads();
  return s;
}

// cos and sin of the rotary angle pos * base^(-2i/d). The angle is formed
// and reduced to [-1/2, 1/2] revolution in double precision; the hardware
// sine/cosine (argument in revolutions) then evaluates the small angle.
__device__ __forceinline__ void rope_angle(int pos, int i, int d, float base, float& c, float& s) {
  const double inv_freq = exp2(-2.0 * static_cast<double>(i) / static_cast<double>(d) *
                               log2(static_cast<double>(base)));
  double rev = static_cast<double>(pos) * inv_freq * 0.15915494309189535;  // 1 / (2 pi)
  rev -= rint(rev);
  const float r = static_cast<float>(rev);
  s = __builtin_amdgcn_sinf(r);
  c = __builtin_amdgcn_cosf(r);
}

// ---- synchronisation words (agent scope: visible across all XCDs) --------
__device__ __forceinline__ unsigned sync_load(const unsigned* p) {
  return __hip_atomic_load(p, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ unsigned sync_add(unsigned* p, unsigned v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void sync_store(unsigned* p, unsigned v) {
  __hip_atomic_store(p, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void sync_or(unsigned* p, unsigned v) {
  __hip_atomic_fetch_or(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace vt
