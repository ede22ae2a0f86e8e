// Device helpers for gfx950 (CDNA4): fp16 packing, wave/block reductions,
// agent-scope synchronisation words.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vt {

constexpr int kWave = 64;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
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

__device__ __forceinline__ u32x4 pack8(const uint16_t (&h)[8]) {
  return u32x4{h[0] | (static_cast<unsigned>(h[1]) << 16), h[2] | (static_cast<unsigned>(h[3]) << 16),
               h[4] | (static_cast<unsigned>(h[5]) << 16), h[6] | (static_cast<unsigned>(h[7]) << 16)};
}

// Raw buffer over [base, base + bytes), bytes < 2^31. A load whose per-lane
// offset is >= bytes returns zero and touches no memory, which gives
// branch-free masked loads (every lane issues, out-of-range lanes cost
// nothing). Only the per-lane offset is range-checked: pass the whole
// offset there and keep the scalar offset 0.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr uint32_t kOOB = 0x80000000u;  // an offset past every buffer

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0),
                                           static_cast<int>(bytes), 0x00020000);
}

__device__ __forceinline__ u32x4 buf_load16(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

// Streaming 16-byte load of weights that are read exactly once per step.
__device__ __forceinline__ u32x4 load_stream(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

__device__ __forceinline__ u32x4 load16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

// DPP move of a float across lanes (ctrl: DPP control word).
template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ float dpp_f(float old, float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, old),
                                                               __builtin_bit_cast(int, v), CTRL,
                                                               ROW_MASK, 0xF, false));
}

// Sum over the 64 lanes of a wave; every lane gets the total. Quad swaps and
// row mirrors give each 16-lane row its sum; the row broadcasts of lane 15
// and lane 31 accumulate the rows into lane 63, which is then read out.
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f<0xB1>(0.f, v);         // quad_perm [1,0,3,2]
  v += dpp_f<0x4E>(0.f, v);         // quad_perm [2,3,0,1]
  v += dpp_f<0x141>(0.f, v);        // row_half_mirror
  v += dpp_f<0x140>(0.f, v);        // row_mirror
  v += dpp_f<0x142, 0xA>(0.f, v);   // row_bcast:15 into rows 1 and 3
  v += dpp_f<0x143, 0xC>(0.f, v);   // row_bcast:31 into rows 2 and 3
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

// Maximum over the 64 lanes of a wave; every lane gets it (same DPP pattern
// as wave_sum; -inf is the identity, so masked-off rows add nothing).
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f<0xB1>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x4E>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x141>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x140>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x142, 0xA>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x143, 0xC>(-INFINITY, v));
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

// Sum over groups of ``width`` consecutive lanes; every lane of a group gets
// the group's sum. Widths 8 and 16 use DPP within a row (quad swaps, then
// the half-row and row mirrors); other powers of two <= 64 use lane shuffles.
__device__ __forceinline__ float group_sum(float v, int width) {
  if (width == 8 || width == 16) {
    v += dpp_f<0xB1>(0.f, v);    // quad_perm [1,0,3,2]
    v += dpp_f<0x4E>(0.f, v);    // quad_perm [2,3,0,1]
    v += dpp_f<0x141>(0.f, v);   // row_half_mirror: the other quad of the half-row
    if (width == 16) v += dpp_f<0x140>(0.f, v);  // row_mirror: the other half-row
    return v;
  }
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

// ---- data shared between workgroups of one launch ---------------------------
// Agent-scope relaxed atomic stores and loads are performed at the level that
// all XCDs share (they bypass each XCD's non-coherent L2). Data that one
// workgroup writes and another reads within a launch moves only through
// them, so a grid barrier needs no L2 writeback or invalidate: the writer
// waits for its stores to complete, then bumps a counter.
__device__ __forceinline__ void st_shared(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ float ld_shared(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The same agent-scope coherent loads (cache policy sc1, as a relaxed
// agent-scope atomic load compiles to) through a buffer resource: an offset
// past the buffer reads zero with no memory traffic, so lanes with nothing to
// load need neither a branch nor a clamped (and then shared, hot) address.
// The 8-byte result is split from the whole 64 bits: bit-casting one element
// of the returned ext-vector makes this compiler reuse element 0.
constexpr int kCoherent = 16;  // sc1

__device__ __forceinline__ void buf_ld_shared2(rsrc_t r, uint32_t off, float& a, float& b) {
  const uint64_t w =
      __builtin_bit_cast(uint64_t, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kCoherent));
  a = __builtin_bit_cast(float, static_cast<uint32_t>(w));
  b = __builtin_bit_cast(float, static_cast<uint32_t>(w >> 32));
}

__device__ __forceinline__ float buf_ld_shared(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kCoherent));
}

// An fp16 value shared between workgroups of one launch (same agent-scope
// coherent path as st_shared / ld_shared).
__device__ __forceinline__ void st_h16_shared(uint16_t* p, uint16_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint16_t ld_h16_shared(const uint16_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Two consecutive floats (8-byte aligned) written by other workgroups.
__device__ __forceinline__ void ld_shared2(const float* p, float& a, float& b) {
  const uint64_t v = __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
  a = __builtin_bit_cast(float, static_cast<uint32_t>(v));
  b = __builtin_bit_cast(float, static_cast<uint32_t>(v >> 32));
}

// Workgroup barrier that orders LDS accesses only: global loads still in
// flight stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Wait for all of this wave's outstanding memory operations (stores
// included) to complete.
__device__ __forceinline__ void mem_done() { __builtin_amdgcn_s_waitcnt(0); }

// ---- synchronisation words (agent scope: visible across all XCDs) --------
// Relaxed: the data they guard moves through st_shared / ld_shared.
__device__ __forceinline__ void sync_store(unsigned* p, unsigned v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void sync_or(unsigned* p, unsigned v) {
  __hip_atomic_fetch_or(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace vt
