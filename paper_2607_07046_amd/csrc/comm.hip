// Transmission-precision scaling of a shard's partial sums (paper Sec. 4.3.2,
// Communication Scaling): to cut the bytes sent to the aggregating device,
// the partial sums are sent in blocks of 32 at FP16, INT8 or INT4 (symmetric
// block-absmax scale) or not at all, the precisions lowered in ascending
// order of importance until the message fits a byte budget (the
// importance-ordered lowering of Sec. 4.2.2). The receiver reconstructs the
// values and adds them to its own sum.
//
// Message layout: blocks in index order, block b at offsets[b]; the block
// format and quantiser are in comm_block.hpp.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <numeric>
#include <vector>

#include "comm_block.hpp"
#include "device.hpp"
#include "internal.hpp"

namespace vt {
namespace comm {

constexpr int BLK = 32;
constexpr int CT = 256;  // threads per workgroup: 8 blocks (one per half-wave)

__host__ __device__ __forceinline__ int block_bytes(int level) { return comm_block_bytes(level); }

// One half-wave per block. Every lane takes part in the shuffles (blocks past
// the end act as pruned); every store goes through the message's buffer
// range and an explicit bound, so no plan content can write outside it.
__global__ void __launch_bounds__(CT) encode_kernel(const uint16_t* p, int nblk, const uint8_t* prec,
                                                    const int32_t* offsets, uint8_t* msg,
                                                    uint32_t msg_bytes) {
  const int b = blockIdx.x * (CT / BLK) + threadIdx.x / BLK;
  const int i = threadIdx.x % BLK;
  const bool valid = b < nblk;
  const int level = valid ? prec[b] : VT_PREC_PRUNED;
  const int64_t o = valid ? offsets[b] : 0;
  const uint16_t raw = valid ? p[static_cast<int64_t>(b) * BLK + i] : 0;
  comm_encode_block_lanes(raw, i, level, o, make_rsrc(msg, msg_bytes), msg_bytes);
}

// out[i] = fp16(base[i] + value[i]) with value = code * s (fp32 multiply,
// then fp32 add: no fused multiply-add, so the rounding steps are fixed).
__global__ void __launch_bounds__(CT) decode_add_kernel(const uint8_t* msg, uint32_t msg_bytes, int n,
                                                        const uint8_t* prec, const int32_t* offsets,
                                                        const uint16_t* base, uint16_t* out) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * CT + threadIdx.x;
  if (i >= n) return;
  const int b = static_cast<int>(i / BLK), j = static_cast<int>(i % BLK);
  const int level = prec[b];
  const int64_t o = offsets[b];
  const rsrc_t rm = make_rsrc(msg, msg_bytes);
  auto at = [&](int64_t off, int len) -> uint32_t {
    return (o >= 0 && off + len <= static_cast<int64_t>(msg_bytes)) ? static_cast<uint32_t>(off) : kOOB;
  };
  float v = 0.f;
  if (level == VT_PREC_FP16) {
    v = h2f(__builtin_amdgcn_raw_buffer_load_b16(rm, at(o + 2 * j, 2), 0, 0));
  } else if (level == VT_PREC_INT8 || level == VT_PREC_INT4) {
    const float s = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rm, at(o, 4), 0, 0));
    int c;
    if (level == VT_PREC_INT8) {
      c = static_cast<int8_t>(__builtin_amdgcn_raw_buffer_load_b8(rm, at(o + 4 + j, 1), 0, 0));
    } else {
      const int byte = __builtin_amdgcn_raw_buffer_load_b8(rm, at(o + 4 + j / 2, 1), 0, 0);
      const int nib = (j & 1) ? (byte >> 4) & 0xF : byte & 0xF;
      c = nib >= 8 ? nib - 16 : nib;
    }
    v = __fmul_rn(static_cast<float>(c), s);
  }
  out[i] = f2h(__fadd_rn(base ? h2f(base[i]) : 0.f, v));
}

}  // namespace comm
}  // namespace vt

using namespace vt;

extern "C" vt_status vt_qplan(const float* importance, int32_t n_blocks, int64_t budget_bytes,
                              uint8_t* prec, int32_t* offsets, int64_t* total_bytes) {
  clear_error();
  if (!importance || !prec || !offsets || !total_bytes) return fail(VT_ERR_ARG, "null argument");
  if (n_blocks < 1 || n_blocks > (1 << 24))
    return fail(VT_ERR_ARG, "n_blocks %d outside 1..2^24", n_blocks);
  for (int b = 0; b < n_blocks; ++b)
    if (!std::isfinite(importance[b])) return fail(VT_ERR_ARG, "importance[%d] is not finite", b);
  std::vector<int> order(n_blocks);
  std::iota(order.begin(), order.end(), 0);
  // ascending importance, the lower block index first on ties
  std::stable_sort(order.begin(), order.end(),
                   [&](int a, int b) { return importance[a] < importance[b]; });
  std::vector<uint8_t> lv(n_blocks, VT_PREC_FP16);
  int64_t total = static_cast<int64_t>(n_blocks) * comm::block_bytes(VT_PREC_FP16);
  // the least lowering that fits: each level down in importance order
  for (int from = VT_PREC_FP16; from < VT_PREC_PRUNED && total > budget_bytes; ++from) {
    for (int b : order) {
      if (total <= budget_bytes) break;
      if (lv[b] == from) {
        total -= comm::block_bytes(from) - comm::block_bytes(from + 1);
        lv[b] = static_cast<uint8_t>(from + 1);
      }
    }
  }
  int64_t acc = 0;
  for (int b = 0; b < n_blocks; ++b) {
    prec[b] = lv[b];
    offsets[b] = static_cast<int32_t>(acc);
    acc += comm::block_bytes(lv[b]);
  }
  *total_bytes = acc;
  return VT_OK;
}

static vt_status check_comm(int32_t n, const void* prec, const void* offsets, const void* msg,
                            size_t msg_bytes) {
  if (n < comm::BLK || n % comm::BLK)
    return fail(VT_ERR_ARG, "n %d is not a positive multiple of %d", n, comm::BLK);
  if (!prec || !offsets || !msg) return fail(VT_ERR_ARG, "null plan or message");
  if (!aligned16(prec) || !aligned16(offsets) || !aligned16(msg))
    return fail(VT_ERR_ALIGN, "plan or message not 16-byte aligned");
  if (msg_bytes >= static_cast<size_t>(kMaxBufferBytes))
    return fail(VT_ERR_UNSUPPORTED, "message of %zu bytes exceeds 2 GiB", msg_bytes);
  return VT_OK;
}

extern "C" vt_status vt_partial_encode(const void* p, int32_t n, const uint8_t* prec,
                                       const int32_t* offsets, void* msg, size_t msg_bytes,
                                       void* stream) {
  clear_error();
  if (!p) return fail(VT_ERR_ARG, "null partial");
  if (!aligned16(p)) return fail(VT_ERR_ALIGN, "partial not 16-byte aligned");
  vt_status st = check_comm(n, prec, offsets, msg, msg_bytes);
  if (st != VT_OK) return st;
  const int nblk = n / comm::BLK;
  const int grid = (nblk + comm::CT / comm::BLK - 1) / (comm::CT / comm::BLK);
  hipLaunchKernelGGL(comm::encode_kernel, dim3(grid), dim3(comm::CT), 0, static_cast<hipStream_t>(stream),
                     static_cast<const uint16_t*>(p), nblk, prec, offsets, static_cast<uint8_t*>(msg),
                     static_cast<uint32_t>(msg_bytes));
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? VT_OK : fail(VT_ERR_HIP, "encode launch: %s", hipGetErrorString(e));
}

extern "C" vt_status vt_partial_decode_add(const void* msg, size_t msg_bytes, int32_t n,
                                           const uint8_t* prec, const int32_t* offsets,
                                           const void* base, void* out, void* stream) {
  clear_error();
  if (!out) return fail(VT_ERR_ARG, "null output");
  if (!aligned16(out) || (base && !aligned16(base)))
    return fail(VT_ERR_ALIGN, "base or output not 16-byte aligned");
  vt_status st = check_comm(n, prec, offsets, msg, msg_bytes);
  if (st != VT_OK) return st;
  const int grid = (n + comm::CT - 1) / comm::CT;
  hipLaunchKernelGGL(comm::decode_add_kernel, dim3(grid), dim3(comm::CT), 0, static_cast<hipStream_t>(stream),
                     static_cast<const uint8_t*>(msg), static_cast<uint32_t>(msg_bytes), n, prec, offsets,
                     static_cast<const uint16_t*>(base), static_cast<uint16_t*>(out));
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? VT_OK : fail(VT_ERR_HIP, "decode launch: %s", hipGetErrorString(e));
}
