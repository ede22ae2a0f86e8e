// Quantisation of one block of 32 partial sums into the transmission
// message (paper Sec. 4.3.2, Communication Scaling), as a collective of the
// 32 lanes of a half-wave: lane i holds element i. Shared by the standalone
// encoder (vt_partial_encode) and the decode epilogues that emit the message
// (vt_layer_decode_emit), so both write the same bytes.
//
// Block wire format at byte offset o of the message:
//   FP16   64 B: the 32 fp16 values
//   INT8   36 B: fp32 scale s, 32 int8 codes           value = code * s
//   INT4   20 B: fp32 scale s, 16 bytes of two 4-bit two's-complement codes,
//                element 2k in the low nibble of byte k
//   PRUNED  0 B
// s = absmax / Q (fp32 division; Q = 127 or 7), code = clamp(rint(x / s),
// -Q, Q) with x / s an fp32 division and rint rounding half to even; an
// all-zero block has s = 0 and codes 0.
#pragma once

#include <hip/hip_runtime.h>

#include "device.hpp"
#include "voltron.h"

namespace vt {

__host__ __device__ __forceinline__ int comm_block_bytes(int level) {
  return level == VT_PREC_FP16 ? 64 : level == VT_PREC_INT8 ? 36 : level == VT_PREC_INT4 ? 20 : 0;
}

// Every lane of the half-wave takes part (the shuffles read the other lanes'
// values); ``raw`` is this lane's fp16 element, ``i`` its index in the block.
// Every store goes through the message's buffer resource and an explicit
// bound, so no plan content writes outside [msg, msg + msg_bytes).
__device__ __forceinline__ void comm_encode_block_lanes(uint16_t raw, int i, int level, int64_t o,
                                                        rsrc_t rm, uint32_t msg_bytes) {
  const float x = h2f(raw);
  float a = fabsf(x);
#pragma unroll
  for (int m = 1; m < 32; m <<= 1) a = fmaxf(a, __shfl_xor(a, m, kWave));  // stays in the half-wave
  const float qm = level == VT_PREC_INT8 ? 127.f : 7.f;
  const float s = __fdiv_rn(a, qm);
  float c = a == 0.f ? 0.f : __builtin_rintf(__fdiv_rn(x, s));
  c = fminf(fmaxf(c, -qm), qm);
  const int ci = static_cast<int>(c);
  const int next = __shfl_down(ci, 1, kWave);  // the odd neighbour's code (INT4 packing)
  auto at = [&](int64_t off, int len) -> uint32_t {  // kOOB unless [off, off + len) fits
    return (o >= 0 && off + len <= static_cast<int64_t>(msg_bytes)) ? static_cast<uint32_t>(off) : kOOB;
  };
  if (level == VT_PREC_FP16) {
    __builtin_amdgcn_raw_buffer_store_b16(raw, rm, at(o + 2 * i, 2), 0, 0);
  } else if (level == VT_PREC_INT8 || level == VT_PREC_INT4) {
    if (i == 0) __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, s), rm, at(o, 4), 0, 0);
    if (level == VT_PREC_INT8) {
      __builtin_amdgcn_raw_buffer_store_b8(static_cast<uint8_t>(ci & 0xFF), rm, at(o + 4 + i, 1), 0, 0);
    } else if ((i & 1) == 0) {
      const uint8_t byte = static_cast<uint8_t>((ci & 0xF) | ((next & 0xF) << 4));
      __builtin_amdgcn_raw_buffer_store_b8(byte, rm, at(o + 4 + i / 2, 1), 0, 0);
    }
  }
}

}  // namespace vt
