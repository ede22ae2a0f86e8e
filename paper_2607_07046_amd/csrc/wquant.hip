// Block quantisation of a shard's weight rows to INT8 / INT4 (paper Sec.
// 2.2 precision heterogeneity, Sec. 4.2.2 importance-aware mixed
// precision, Sec. 4.3.1 precision scaling): the format the decode kernel
// reads through vt_layer_decode_q.
//
// Per row, blocks of 32 consecutive columns (the last may be partial; its
// missing columns count as zero). Block scale s = fp16(absmax / Q) (fp32
// division, round to nearest even; Q = 127 or 7); codes c = clamp(rint(w /
// s), -Q, Q) with w and s as fp32 and the division in fp32 (ties to even);
// s = 0 gives c = 0. INT8 codes are bytes in column order; INT4 codes are
// nibbles c + 8, 8 columns per 4 bytes: column 8g + i (i < 4) in the low
// nibble of byte 4g + i, column 8g + 4 + i in its high nibble.
#include <hip/hip_runtime.h>

#include "device.hpp"
#include "internal.hpp"

namespace vt {
namespace wq {

constexpr int QT = 256;  // threads per workgroup, one block of 32 columns each

__global__ void __launch_bounds__(QT) quantize_kernel(const uint16_t* __restrict__ w, int64_t ld, int rows,
                                                      int cols, int prec, uint8_t* __restrict__ codes,
                                                      int64_t ld_codes, uint16_t* __restrict__ scales,
                                                      int64_t ld_scales) {
  const int nb = (cols + 31) / 32;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * QT + threadIdx.x;
  if (i >= static_cast<int64_t>(rows) * nb) return;
  const int r = static_cast<int>(i / nb), b = static_cast<int>(i % nb);
  const int n = min(32, cols - b * 32);
  const uint16_t* src = w + r * ld + b * 32;
  float v[32];
  float a = 0.f;
#pragma unroll
  for (int e = 0; e < 32; ++e) {
    v[e] = e < n ? h2f(src[e]) : 0.f;
    a = fmaxf(a, fabsf(v[e]));
  }
  const float qm = prec == VT_W_INT8 ? 127.f : 7.f;
  const uint16_t s16 = f2h(__fdiv_rn(a, qm));
  const float s = h2f(s16);
  int c[32];
#pragma unroll
  for (int e = 0; e < 32; ++e)
    c[e] = s > 0.f ? static_cast<int>(fminf(fmaxf(__builtin_rintf(__fdiv_rn(v[e], s)), -qm), qm)) : 0;
  scales[r * ld_scales + b] = s16;
  if (prec == VT_W_INT8) {
    uint32_t word[8];
#pragma unroll
    for (int k = 0; k < 8; ++k)
      word[k] = (c[4 * k] & 0xFF) | ((c[4 * k + 1] & 0xFF) << 8) | ((c[4 * k + 2] & 0xFF) << 16) |
                (static_cast<uint32_t>(c[4 * k + 3] & 0xFF) << 24);
    u32x4* dst = reinterpret_cast<u32x4*>(codes + r * ld_codes + b * 32);
    dst[0] = u32x4{word[0], word[1], word[2], word[3]};
    dst[1] = u32x4{word[4], word[5], word[6], word[7]};
  } else {
    uint32_t word[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      uint32_t x = 0;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint32_t byte = static_cast<uint32_t>(c[8 * g + k] + 8) | (static_cast<uint32_t>(c[8 * g + 4 + k] + 8) << 4);
        x |= byte << (8 * k);
      }
      word[g] = x;
    }
    *reinterpret_cast<u32x4*>(codes + r * ld_codes + b * 16) = u32x4{word[0], word[1], word[2], word[3]};
  }
}

}  // namespace wq
}  // namespace vt

using namespace vt;

extern "C" vt_status vt_quantize_rows(const void* w, int64_t ld, int32_t rows, int32_t cols, int32_t prec,
                                      void* codes, int64_t ld_codes, void* scales, int64_t ld_scales,
                                      void* stream) {
  clear_error();
  if (prec != VT_W_INT8 && prec != VT_W_INT4)
    return fail(VT_ERR_ARG, "precision %d is neither VT_W_INT8 nor VT_W_INT4", prec);
  if (rows < 0 || cols < 1) return fail(VT_ERR_ARG, "rows %d / cols %d invalid", rows, cols);
  if (rows == 0) return VT_OK;
  if (!w || !codes || !scales) return fail(VT_ERR_ARG, "null buffer");
  if (!aligned16(w) || !aligned16(codes)) return fail(VT_ERR_ALIGN, "weights or codes not 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(scales) % 2) return fail(VT_ERR_ALIGN, "scales not 2-byte aligned");
  const int64_t nb = (cols + 31) / 32;
  const int64_t need = nb * (prec == VT_W_INT8 ? 32 : 16);
  if (ld < cols || ld % 8) return fail(VT_ERR_ARG, "ld %lld must be a multiple of 8 and >= cols %d",
                                       static_cast<long long>(ld), cols);
  if (ld_codes < need || ld_codes % 16)
    return fail(VT_ERR_ARG, "ld_codes %lld must be a multiple of 16 and >= %lld",
                static_cast<long long>(ld_codes), static_cast<long long>(need));
  if (ld_scales < nb)
    return fail(VT_ERR_ARG, "ld_scales %lld < %lld blocks", static_cast<long long>(ld_scales),
                static_cast<long long>(nb));
  const int64_t items = static_cast<int64_t>(rows) * nb;
  if (items > (int64_t(1) << 31) - wq::QT) return fail(VT_ERR_UNSUPPORTED, "%lld blocks", static_cast<long long>(items));
  const int grid = static_cast<int>((items + wq::QT - 1) / wq::QT);
  hipLaunchKernelGGL(wq::quantize_kernel, dim3(grid), dim3(wq::QT), 0, static_cast<hipStream_t>(stream),
                     static_cast<const uint16_t*>(w), ld, rows, cols, prec, static_cast<uint8_t*>(codes),
                     ld_codes, static_cast<uint16_t*>(scales), ld_scales);
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? VT_OK : fail(VT_ERR_HIP, "quantize launch: %s", hipGetErrorString(e));
}
