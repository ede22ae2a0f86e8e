// Elastic re-partition (paper Sec. 4.3.1): when the partition changes, a
// device gathers its new shard's weights out of the layer's full weights
// and takes over the KV heads its new shard owns. Shards are allocated
// separately (Sec. 4.3.1, Overhead Mitigation), so a new shard is packed
// into new buffers on a second stream while decode continues on the old
// ones. Pure data movement: every value is copied bit for bit.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "device.hpp"
#include "internal.hpp"

namespace vt {
namespace rp {

constexpr int CT = 256;

// dst[r][c] = src[r][c0 + c] for c < cols and 0 for cols <= c < dcols
// (fp16, strides in elements; dst rows and dcols in whole 8-element chunks
// of 16 bytes). A chunk's 8 source elements are one 16-byte load when the
// source chunk is 16-byte aligned (ALIGNED), else 8 two-byte loads.
template <bool ALIGNED>
__global__ void __launch_bounds__(CT) copy2d_kernel(const uint16_t* __restrict__ src, int64_t lds, int64_t c0,
                                                    uint16_t* __restrict__ dst, int64_t ldd, int rows, int cols,
                                                    int dcols) {
  const int nch = dcols / 8;
  const int64_t total = static_cast<int64_t>(rows) * nch;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * CT + threadIdx.x; i < total;
       i += static_cast<int64_t>(gridDim.x) * CT) {
    const int r = static_cast<int>(i / nch), ch = static_cast<int>(i % nch);
    const int c = ch * 8;
    const uint16_t* s = src + r * lds + c0 + c;
    u32x4 v;
    if (ALIGNED && c + 8 <= cols) {
      v = *reinterpret_cast<const u32x4*>(s);
    } else {
      uint16_t h[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) h[e] = c + e < cols ? s[e] : 0;
      v = pack8(h);
    }
    *reinterpret_cast<u32x4*>(dst + r * ldd + c) = v;
  }
}

static vt_status copy2d(const uint16_t* src, int64_t lds, int64_t c0, uint16_t* dst, int64_t ldd, int rows, int cols,
                        int dcols, hipStream_t s) {
  if (rows <= 0 || dcols <= 0) return VT_OK;
  const int64_t chunks = static_cast<int64_t>(rows) * (dcols / 8);
  const int grid = static_cast<int>(std::min<int64_t>((chunks + CT - 1) / CT, 8192));
  if (c0 % 8 == 0)
    hipLaunchKernelGGL(copy2d_kernel<true>, dim3(grid), dim3(CT), 0, s, src, lds, c0, dst, ldd, rows, cols, dcols);
  else
    hipLaunchKernelGGL(copy2d_kernel<false>, dim3(grid), dim3(CT), 0, s, src, lds, c0, dst, ldd, rows, cols, dcols);
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? VT_OK : fail(VT_ERR_HIP, "copy launch: %s", hipGetErrorString(e));
}

}  // namespace rp
}  // namespace vt

using namespace vt;

namespace {

// A matrix argument: rows x row length (elements) at stride ld.
vt_status check_mat(const void* p, int64_t ld, int64_t rowlen, int64_t rows, const char* what) {
  if (rows == 0 || rowlen == 0) return VT_OK;
  if (!p) return fail(VT_ERR_ARG, "%s is NULL", what);
  if (!aligned16(p)) return fail(VT_ERR_ALIGN, "%s is not 16-byte aligned", what);
  if (ld < rowlen || ld % 8)
    return fail(VT_ERR_ARG, "ld of %s (%lld) must be a multiple of 8 and >= %lld", what,
                static_cast<long long>(ld), static_cast<long long>(rowlen));
  return VT_OK;
}

}  // namespace

extern "C" vt_status vt_shard_pack(const vt_shard_spec* spec, const vt_layer_weights* full,
                                   const vt_layer_weights* out, void* stream) {
  clear_error();
  if (!spec || !full || !out) return fail(VT_ERR_ARG, "null argument");
  const vt_layer_dims& D = spec->dims;
  const vt_shard_info& in = spec->info;
  const int64_t H = D.hidden, d = D.head_dim, F = D.ffn;
  const int64_t nqd = static_cast<int64_t>(D.n_heads) * d, nkd = static_cast<int64_t>(D.n_kv_heads) * d;
  const int64_t qd = static_cast<int64_t>(in.n_q_heads) * d, kd = static_cast<int64_t>(in.n_kv_heads) * d;
  const int64_t q0 = static_cast<int64_t>(in.q_head_begin) * d, k0 = static_cast<int64_t>(in.kv_head_begin) * d;
  const int64_t nc = in.n_cols, c0 = in.col_begin;
  const int64_t ncp = (nc + 7) / 8 * 8;  // the shard's Wd rows: n_cols rounded up to 8, zero past n_cols
  vt_status st;
  struct M {
    const void* p;
    int64_t ld, rowlen, rows;
    const char* what;
  };
  const M checks[] = {
      {full->g_attn, H, H, 1, "full g_attn"}, {full->g_ffn, H, H, 1, "full g_ffn"},
      {full->wq, full->ld_q, H, nqd, "full wq"}, {full->wk, full->ld_k, H, nkd, "full wk"},
      {full->wv, full->ld_v, H, nkd, "full wv"}, {full->wo, full->ld_o, nqd, H, "full wo"},
      {full->wg, full->ld_g, H, F, "full wg"},   {full->wu, full->ld_u, H, F, "full wu"},
      {full->wd, full->ld_d, F, H, "full wd"},   {out->g_attn, H, H, 1, "g_attn"},
      {out->g_ffn, H, H, 1, "g_ffn"},            {out->wq, out->ld_q, H, qd, "wq"},
      {out->wk, out->ld_k, H, kd, "wk"},         {out->wv, out->ld_v, H, kd, "wv"},
      {out->wo, out->ld_o, qd, H, "wo"},         {out->wg, out->ld_g, H, nc, "wg"},
      {out->wu, out->ld_u, H, nc, "wu"},         {out->wd, out->ld_d, ncp, H, "wd"},
  };
  for (const M& m : checks)
    if ((st = check_mat(m.p, m.ld, m.rowlen, m.rows, m.what)) != VT_OK) return st;
  for (const M& m : checks)
    if (m.rows * m.ld * 2 >= (int64_t(1) << 40))
      return fail(VT_ERR_UNSUPPORTED, "%s is implausibly large", m.what);
  hipStream_t s = static_cast<hipStream_t>(stream);
  auto h = [](const void* p) { return static_cast<const uint16_t*>(p); };
  auto o = [](const void* p) { return static_cast<uint16_t*>(const_cast<void*>(p)); };
  if ((st = rp::copy2d(h(full->g_attn), H, 0, o(out->g_attn), H, 1, H, H, s)) != VT_OK) return st;
  if ((st = rp::copy2d(h(full->g_ffn), H, 0, o(out->g_ffn), H, 1, H, H, s)) != VT_OK) return st;
  if (qd > 0) {
    if ((st = rp::copy2d(h(full->wq) + q0 * full->ld_q, full->ld_q, 0, o(out->wq), out->ld_q, qd, H, H, s)) != VT_OK)
      return st;
    if ((st = rp::copy2d(h(full->wk) + k0 * full->ld_k, full->ld_k, 0, o(out->wk), out->ld_k, kd, H, H, s)) != VT_OK)
      return st;
    if ((st = rp::copy2d(h(full->wv) + k0 * full->ld_v, full->ld_v, 0, o(out->wv), out->ld_v, kd, H, H, s)) != VT_OK)
      return st;
    // Wo: the shard's columns; its rows are whole 8-element chunks since qd is
    if ((st = rp::copy2d(h(full->wo), full->ld_o, q0, o(out->wo), out->ld_o, H, qd, qd, s)) != VT_OK) return st;
  }
  if (nc > 0) {
    if ((st = rp::copy2d(h(full->wg) + c0 * full->ld_g, full->ld_g, 0, o(out->wg), out->ld_g, nc, H, H, s)) != VT_OK)
      return st;
    if ((st = rp::copy2d(h(full->wu) + c0 * full->ld_u, full->ld_u, 0, o(out->wu), out->ld_u, nc, H, H, s)) != VT_OK)
      return st;
    if ((st = rp::copy2d(h(full->wd), full->ld_d, c0, o(out->wd), out->ld_d, H, nc, ncp, s)) != VT_OK) return st;
  }
  return VT_OK;
}

extern "C" vt_status vt_kv_copy_heads(const vt_kv_view* src, int32_t src_head0, const vt_kv_view* dst,
                                      int32_t dst_head0, int32_t n_heads, int32_t n_pos, void* stream) {
  clear_error();
  if (!src || !dst) return fail(VT_ERR_ARG, "null KV view");
  if (n_heads < 0 || n_pos < 0) return fail(VT_ERR_ARG, "n_heads %d / n_pos %d < 0", n_heads, n_pos);
  if (n_heads == 0 || n_pos == 0) return VT_OK;
  if (src->head_dim != dst->head_dim || (src->head_dim != 64 && src->head_dim != 128))
    return fail(VT_ERR_ARG, "head_dim %d vs %d", src->head_dim, dst->head_dim);
  if (src_head0 < 0 || dst_head0 < 0 || src_head0 + static_cast<int64_t>(n_heads) > src->n_kv_heads ||
      dst_head0 + static_cast<int64_t>(n_heads) > dst->n_kv_heads)
    return fail(VT_ERR_ARG, "head range outside a cache (%d+%d of %d, %d+%d of %d)", src_head0, n_heads,
                src->n_kv_heads, dst_head0, n_heads, dst->n_kv_heads);
  if (n_pos > src->capacity || n_pos > dst->capacity)
    return fail(VT_ERR_ARG, "n_pos %d exceeds a capacity (%d, %d)", n_pos, src->capacity, dst->capacity);
  if (!src->k || !src->v || !dst->k || !dst->v) return fail(VT_ERR_ARG, "null cache buffer");
  if (!aligned16(src->k) || !aligned16(src->v) || !aligned16(dst->k) || !aligned16(dst->v))
    return fail(VT_ERR_ALIGN, "cache buffers must be 16-byte aligned");
  const int64_t d = src->head_dim;
  const int64_t lds = static_cast<int64_t>(src->capacity) * d, ldd = static_cast<int64_t>(dst->capacity) * d;
  const int cols = static_cast<int>(n_pos * d);
  hipStream_t s = static_cast<hipStream_t>(stream);
  vt_status st;
  const uint16_t* sk = static_cast<const uint16_t*>(src->k) + src_head0 * lds;
  const uint16_t* sv = static_cast<const uint16_t*>(src->v) + src_head0 * lds;
  uint16_t* dk = static_cast<uint16_t*>(dst->k) + dst_head0 * ldd;
  uint16_t* dv = static_cast<uint16_t*>(dst->v) + dst_head0 * ldd;
  if ((st = rp::copy2d(sk, lds, 0, dk, ldd, n_heads, cols, cols, s)) != VT_OK) return st;
  return rp::copy2d(sv, lds, 0, dv, ldd, n_heads, cols, cols, s);
}
