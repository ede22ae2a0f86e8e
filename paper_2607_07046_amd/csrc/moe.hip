// Mixture-of-experts FFN of a shard on gfx950 (paper Sec. 2.1 FFN variants;
// the MoE model of Table 3), batch-1 decode: one persistent launch of one
// 512-thread workgroup per CU runs the router GEMV, the routing (in every
// workgroup, from the logits), the selected experts' gate/up GEMV and their
// down GEMV, separated by grid barriers, on the GEMV machinery of the dense
// decode kernel.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "device.hpp"
#include "gemv.hpp"
#include "internal.hpp"

namespace vt {
namespace dec {

// ---------------------------------------------------------------------------
// Mixture-of-experts FFN of a shard (paper Sec. 2.1 FFN variants; the MoE
// model of Table 3): w = RMSNorm(h) * g_ffn; router logits Wr w over the E
// experts; the top_k largest (ties: lower index) with their softmax
// probabilities p (over all E); output sum over the selected experts of
// p_e Wd_e (silu(Wg_e w) * (Wu_e w)), over this shard's columns of every
// expert. One persistent launch: router GEMV | routing (every workgroup,
// from the logits) + the selected experts' gate/up GEMV | down GEMV.
// ---------------------------------------------------------------------------
constexpr int MOE_MAX_E = 256, MOE_MAX_K = 8;
// (the sync words sit at the start of the workspace, as for decode)
static_assert(SW_ERR * 4 == VT_WS_ERROR_WORD, "the error word's documented offset");

struct MoeParams {
  int H, E, topk, ncols, npe;  // npe: a slot's share of the down input, whole 512-column segments
  uint64_t m_ncols;            // div_m40 multiplier of ncols
  float eps;
  const uint16_t *g_ffn, *h, *peer_f;
  const uint8_t *wr, *wg, *wu, *wd;  // strides in bytes
  int64_t ld_r, ld_g, ld_u, ld_d;
  uint16_t *p_ffn, *y;
  float *logits, *m;  // m: [topk][ncols]
  int32_t* sel_out;
  float* prob_out;
  unsigned* sync;
};

// q / n for 0 <= q < 2^18 and n < 2^15 with m = floor(2^40 / n) + 1 (exact
// while q * n < 2^40).
__device__ __forceinline__ int div_m40(int q, uint64_t m) {
  return static_cast<int>((static_cast<uint64_t>(static_cast<uint32_t>(q)) * m) >> 40);
}

// The selected experts (each < 256) packed a byte per slot into one
// wave-uniform 64-bit word: a slot's expert is a shift and a mask in scalar
// registers (a register array indexed by the slot would be placed in
// scratch memory).
__device__ __forceinline__ int slot_expert(uint64_t sel8, int sl) {
  return static_cast<int>((sel8 >> (8 * sl)) & 0xFFu);
}

// Virtual row 2u (+1): the gate (up) row of column j of the expert in slot
// s, u = s * ncols + j; expert e's column j is row e * ncols + j of wg / wu.
struct RowsMoePair {
  static constexpr bool kSlotTail = false;
  Mat g, u;
  int ncols, topk;
  uint64_t m_ncols;  // div_m40 multiplier of ncols
  uint64_t sel8;
  // (rows past the phase's units are asked for by loads that read nothing;
  // the slot is clamped all the same)
  __device__ __forceinline__ RowAt at(int r) const {
    const int un = r >> 1, sl = min(div_m40(un, m_ncols), topk - 1), j = un - sl * ncols;
    const int row = slot_expert(sel8, sl) * ncols + j;
    return (r & 1) ? mat_row(u, row) : mat_row(g, row);
  }
  __device__ __forceinline__ uint32_t seg_off(int sg) const { return plain_seg(sg); }
};

// Row r of the down projection over the selected experts: its input is the
// slots' m vectors one after the other, each padded to spe segments;
// segment sg of row r is in the matrix of the expert of slot sg / spe
// (expert e's rows start at byte e * H * ld).
struct RowsMoeDown {
  static constexpr bool kSlotTail = true;
  Mat d;
  int H, spe, ncols;
  uint32_t rcp_spe;  // div_rcp reciprocal of spe
  uint64_t sel8;
  __device__ __forceinline__ RowAt at(int r) const { return mat_row(d, r); }
  __device__ __forceinline__ uint32_t seg_off(int sg) const {
    const int sl = div_rcp(sg, rcp_spe), ls = sg - sl * spe;
    return static_cast<uint32_t>(slot_expert(sel8, sl) * H) * d.ld + static_cast<uint32_t>(ls) * 1024u;
  }
  // columns of slot sl's input are [sl * spe * 512, that + ncols)
  __device__ __forceinline__ int col_limit(int sg) const {
    return div_rcp(sg, rcp_spe) * spe * Fmt<FMT_F16>::SEGC + ncols;
  }
};

// Every workgroup: the top_k experts and their probabilities from the E
// logits, into LDS (sel / prob). Expert t's rank is the number of experts
// ordered before it: a larger logit, or an equal one at a lower index. With
// key(t) = (order-preserving bits of the logit, +0 for -0) << 8 | (255 - t)
// that is the number of larger keys, one 64-bit compare per pair. The E x E
// compares are split over all waves (expert t % E64 on every thread, the
// keys in E64 / (NT / E64) long runs, wave-uniform so every key read is an
// LDS broadcast); wave 0 meanwhile takes the softmax maximum and
// denominator. sel entries start at 0, so they name an expert whatever the
// logits hold. ``scr`` is LDS scratch of 1536 floats, 16-byte aligned. Ends
// with a workgroup barrier.
__device__ __forceinline__ uint64_t route_key(float l, int t) {
  const uint32_t b = __float_as_uint(l + 0.0f);  // -0 -> +0: equal logits, equal keys
  const uint32_t o = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
  return (static_cast<uint64_t>(o) << 8) | static_cast<uint64_t>(255 - t);
}

__device__ __forceinline__ void moe_route(const MoeParams& P, float* scr, int* sel, float* prob) {
  uint64_t* key = reinterpret_cast<uint64_t*>(scr);  // [MOE_MAX_E]
  float* lg = scr + 2 * MOE_MAX_E;                    // [MOE_MAX_E] logits, -inf past E
  int* part = reinterpret_cast<int*>(scr + 3 * MOE_MAX_E);  // [NT] partial ranks
  float* stat = scr + 3 * MOE_MAX_E + NT;             // max, denominator
  const int t = threadIdx.x;
  if (t < MOE_MAX_K) {
    sel[t] = 0;
    prob[t] = 0.f;
  }
  if (t < MOE_MAX_E) {
    const uint32_t off = static_cast<uint32_t>(t) * 4u | (static_cast<uint32_t>(t >= P.E) << 31);
    const float l = buf_ld_shared(make_rsrc(P.logits, static_cast<uint32_t>(P.E) * 4u), off);
    lg[t] = t < P.E ? l : -INFINITY;
    key[t] = t < P.E ? route_key(l, t) : 0ull;  // below every expert's key
  }
  __syncthreads();
  const int e64 = (P.E + 63) & ~63;
  const int np = NT / e64, run = e64 / np;
  const int pr = t / e64, te = t - pr * e64;
  if (pr < np) {
    const uint64_t mine = key[te];
    int cnt = 0;
    const int i0 = pr * run;
#pragma unroll 8
    for (int i = 0; i < run; ++i) cnt += key[i0 + i] > mine ? 1 : 0;
    part[pr * e64 + te] = cnt;
  }
  if (t < kWave) {
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < MOE_MAX_E / kWave; ++j) mx = fmaxf(mx, lg[t + kWave * j]);
    mx = wave_max(mx);
    float sm = 0.f;
#pragma unroll
    for (int j = 0; j < MOE_MAX_E / kWave; ++j) sm += __expf(lg[t + kWave * j] - mx);
    sm = wave_sum(sm);
    if (t == 0) {
      stat[0] = mx;
      stat[1] = sm;
    }
  }
  __syncthreads();
  if (t < P.E) {
    int rank = 0;
    for (int q = 0; q < np; ++q) rank += part[q * e64 + t];
    if (rank < P.topk) {
      sel[rank] = t;
      prob[rank] = __expf(lg[t] - stat[0]) / stat[1];
    }
  }
  __syncthreads();
}

// xs[k] for k < topk * npe: slot k / npe's m value at column k % npe, zero
// from ncols on. Coherent loads in batches; positions without a value read
// nothing (offset past the buffer). Ends with a workgroup barrier.
__device__ __forceinline__ void moe_stage_down(const MoeParams& P, uint16_t* xs, uint32_t rcp_spe) {
  constexpr int B = 8;
  const int n = P.topk * P.npe;
  const rsrc_t rm = make_rsrc(P.m, static_cast<uint32_t>(P.topk * P.ncols) * 4u);
  for (int c0 = 0; c0 < n; c0 += B * NT) {
    float v[B];
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int k = c0 + threadIdx.x + u * NT;
      const int sl = div_rcp(k >> 9, rcp_spe), j = k - sl * P.npe;
      const bool ok = k < n && j < P.ncols;
      const uint32_t off = static_cast<uint32_t>(sl * P.ncols + j) * 4u;
      v[u] = buf_ld_shared(rm, off | (static_cast<uint32_t>(!ok) << 31));
    }
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int k = c0 + threadIdx.x + u * NT;
      if (k < n) xs[k] = f2h(v[u]);
    }
  }
  __syncthreads();
}

__global__ void __launch_bounds__(NT) moe_kernel(MoeParams P) {
  extern __shared__ float lds[];
  // LDS: xs | slots[MAX_SLOTS] | red[16] | sel[MOE_MAX_K] | prob[MOE_MAX_K]
  const int kmax = max(padded(P.H, FMT_F16), P.topk * P.npe);
  uint16_t* xs = reinterpret_cast<uint16_t*>(lds);
  float* slots = lds + kmax / 2;
  float* red = slots + MAX_SLOTS;
  int* sel = reinterpret_cast<int*>(red + 16);
  float* prob = reinterpret_cast<float*>(sel + MOE_MAX_K);

  // router logits (xs keeps w for the gate/up phase); h and the gains
  // depend on nothing in this launch, so their loads leave first
  RmsInH<4> hin;
  gemv_phase<1, FMT_F16>(
      RowsOne{make_mat(P.wr, P.ld_r, P.E, nullptr, 0)}, P.E, P.H, xs, slots, nullptr,
      [&]() { hin.load(P.h, P.g_ffn, P.H); },
      [&]() { hin.finish(P.H, padded(P.H, FMT_F16), P.eps, xs, red); },
      [&](int e, const float* v) { st_shared(P.logits + e, v[0]); });
  grid_arrive(P.sync);
  grid_wait(P.sync, 1);
  moe_route(P, slots, sel, prob);  // slots are free between phases
  if (blockIdx.x == 0 && threadIdx.x < P.topk) {
    if (P.sel_out) P.sel_out[threadIdx.x] = sel[threadIdx.x];
    if (P.prob_out) P.prob_out[threadIdx.x] = prob[threadIdx.x];
  }
  // the selected experts' gate/up rows; m = p_e * silu(gate) * up
  uint64_t sel8 = 0;
#pragma unroll
  for (int i = 0; i < MOE_MAX_K; ++i)
    sel8 |= static_cast<uint64_t>(__builtin_amdgcn_readfirstlane(sel[i]) & 0xFF) << (8 * i);
  const RowsMoePair rp{make_mat(P.wg, P.ld_g, static_cast<int64_t>(P.E) * P.ncols, nullptr, 0),
                       make_mat(P.wu, P.ld_u, static_cast<int64_t>(P.E) * P.ncols, nullptr, 0),
                       P.ncols,
                       P.topk,
                       P.m_ncols,
                       sel8};
  const int spe = P.npe / Fmt<FMT_F16>::SEGC;
  const RowsMoeDown rd{make_mat(P.wd, P.ld_d, static_cast<int64_t>(P.E) * P.H, nullptr, 0),
                       P.H,
                       spe,
                       P.ncols,
                       (1u << 24) / static_cast<uint32_t>(spe) + 1u,
                       sel8};
  gemv_phase<2, FMT_F16>(
      rp, P.topk * P.ncols, P.H, xs, slots, nullptr, []() { __syncthreads(); },
      [&](int un, const float* v) {
        const int sl = un / P.ncols;
        const float gt = v[0], up = v[1];
        st_shared(P.m + un, prob[sl] * (gt / (1.0f + __expf(-gt)) * up));
      });
  grid_arrive(P.sync);
  // down rows over the selected experts' columns
  gemv_phase<1, FMT_F16>(
      rd, P.H, P.topk * P.npe, xs, slots, nullptr,
      [&]() {
        grid_wait(P.sync, 2);
        moe_stage_down(P, xs, rd.rcp_spe);
      },
      [&](int r, const float* v) {
        const float pf = v[0];
        P.p_ffn[r] = f2h(pf);
        if (P.y) P.y[r] = f2h(h2f(P.h[r]) + pf + (P.peer_f ? h2f(P.peer_f[r]) : 0.f));
      });
  grid_exit(P.sync);
}

}  // namespace dec
}  // namespace vt

using namespace vt;

namespace {

inline int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

vt_status check_io_vec(const void* p, const char* name, bool required) {
  if (!p) return required ? fail(VT_ERR_ARG, "%s is NULL", name) : VT_OK;
  if (!aligned16(p)) return fail(VT_ERR_ALIGN, "%s is not 16-byte aligned", name);
  return VT_OK;
}

// Per device: CU count and LDS limit, and the MoE kernel's dynamic LDS
// allowance raised to that limit once.
struct MoeDevice {
  int cus = 0;
  size_t max_lds = 0;
};
std::mutex g_moe_mu;
std::vector<MoeDevice> g_moe_dev;

vt_status moe_device(MoeDevice* out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(VT_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  std::lock_guard<std::mutex> lk(g_moe_mu);
  if (static_cast<int>(g_moe_dev.size()) <= dev) g_moe_dev.resize(dev + 1);
  MoeDevice& di = g_moe_dev[dev];
  if (di.cus == 0) {
    int cus = 0, lds = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
    if (e != hipSuccess) return fail(VT_ERR_HIP, "hipDeviceGetAttribute: %s", hipGetErrorString(e));
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(dec::moe_kernel),
                              hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    (void)hipGetLastError();
    di.cus = cus;
    di.max_lds = static_cast<size_t>(lds);
  }
  *out = di;
  return VT_OK;
}

struct MoeWs {
  size_t sync, logits, m, total;
  int npe;
};

MoeWs moe_ws_layout(const vt_shard_spec& s, int32_t top_k, int32_t n_experts) {
  MoeWs w{};
  w.npe = static_cast<int>(std::max<int64_t>(512, round_up(s.info.n_cols, 512)));
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off += static_cast<size_t>(round_up(static_cast<int64_t>(bytes), 256));
    return at;
  };
  w.sync = take(sizeof(unsigned) * (dec::SW_GROUP + dec::SW_GROUP_STRIDE));
  w.logits = take(sizeof(float) * n_experts);
  w.m = take(sizeof(float) * static_cast<size_t>(top_k) * w.npe);
  w.total = off;
  return w;
}

vt_status check_moe_args(const vt_shard_spec* spec, int32_t n_experts, int32_t top_k) {
  if (!spec) return fail(VT_ERR_ARG, "null spec");
  if (n_experts < 1 || n_experts > dec::MOE_MAX_E)
    return fail(VT_ERR_UNSUPPORTED, "n_experts %d outside [1, %d]", n_experts, dec::MOE_MAX_E);
  if (top_k < 1 || top_k > std::min(n_experts, dec::MOE_MAX_K))
    return fail(VT_ERR_ARG, "top_k %d outside [1, min(n_experts, %d)]", top_k, dec::MOE_MAX_K);
  if (spec->info.n_cols >= 32768) return fail(VT_ERR_UNSUPPORTED, "n_cols %d >= 32768", spec->info.n_cols);
  return VT_OK;
}

}  // namespace

extern "C" vt_status vt_moe_workspace_size(const vt_shard_spec* spec, int32_t n_experts, int32_t top_k,
                                           size_t* bytes) {
  clear_error();
  if (!bytes) return fail(VT_ERR_ARG, "null argument");
  vt_status st = check_moe_args(spec, n_experts, top_k);
  if (st != VT_OK) return st;
  *bytes = moe_ws_layout(*spec, top_k, n_experts).total;
  return VT_OK;
}

extern "C" vt_status vt_moe_ffn_decode(const vt_shard_spec* spec, const vt_moe_weights* w, int32_t n_experts,
                                       int32_t top_k, const vt_layer_io* io, int32_t* sel_out, float* prob_out,
                                       void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  vt_status st = check_moe_args(spec, n_experts, top_k);
  if (st != VT_OK) return st;
  if (!w || !io) return fail(VT_ERR_ARG, "null argument");
  const vt_layer_dims& D = spec->dims;
  const int64_t H = D.hidden, E = n_experts, nc = spec->info.n_cols;
  if (H % 8 || H > 16384) return fail(VT_ERR_UNSUPPORTED, "hidden %lld: a multiple of 8 up to 16384", (long long)H);
  if (!w->g_ffn || !aligned16(w->g_ffn)) return fail(VT_ERR_ARG, "g_ffn NULL or not 16-byte aligned");
  struct M {
    const void* p;
    int64_t ld, rowlen, rows;
    const char* what;
  };
  const M mats[] = {{w->wr, w->ld_r, H, E, "wr"},
                    {w->wg, w->ld_g, H, E * nc, "wg"},
                    {w->wu, w->ld_u, H, E * nc, "wu"},
                    {w->wd, w->ld_d, nc, E * H, "wd"}};
  for (const M& m : mats) {
    if (m.rows == 0 || m.rowlen == 0) continue;
    if (!m.p) return fail(VT_ERR_ARG, "%s is NULL", m.what);
    if (!aligned16(m.p)) return fail(VT_ERR_ALIGN, "%s is not 16-byte aligned", m.what);
    if (m.ld < m.rowlen || m.ld % 8)
      return fail(VT_ERR_ARG, "ld of %s (%lld) must be a multiple of 8 and >= %lld", m.what,
                  static_cast<long long>(m.ld), static_cast<long long>(m.rowlen));
    if (m.rows * m.ld * 2 >= (int64_t(1) << 31))
      return fail(VT_ERR_UNSUPPORTED, "%s spans 2 GiB or more", m.what);
  }
  if ((st = check_io_vec(io->h, "h", true)) != VT_OK) return st;
  if ((st = check_io_vec(io->peer_ffn, "peer_ffn", false)) != VT_OK) return st;
  if ((st = check_io_vec(io->ffn_partial, "ffn_partial", true)) != VT_OK) return st;
  if ((st = check_io_vec(io->y, "y", false)) != VT_OK) return st;
  const MoeWs L = moe_ws_layout(*spec, top_k, n_experts);
  if (!ws || ws_bytes < L.total) return fail(VT_ERR_WORKSPACE, "workspace %zu bytes, need %zu", ws_bytes, L.total);
  if (!aligned16(ws)) return fail(VT_ERR_ALIGN, "workspace not 16-byte aligned");
  MoeDevice dv;
  if ((st = moe_device(&dv)) != VT_OK) return st;
  const MoeDevice* di = &dv;

  dec::MoeParams P{};
  P.H = static_cast<int>(H);
  P.E = n_experts;
  P.topk = top_k;
  P.ncols = static_cast<int>(nc);
  P.npe = L.npe;
  P.m_ncols = nc > 0 ? (uint64_t(1) << 40) / static_cast<uint64_t>(nc) + 1 : 1;
  P.eps = D.rms_eps;
  P.g_ffn = static_cast<const uint16_t*>(w->g_ffn);
  P.h = static_cast<const uint16_t*>(io->h);
  P.peer_f = static_cast<const uint16_t*>(io->peer_ffn);
  P.wr = static_cast<const uint8_t*>(w->wr);
  P.wg = nc > 0 ? static_cast<const uint8_t*>(w->wg) : nullptr;
  P.wu = nc > 0 ? static_cast<const uint8_t*>(w->wu) : nullptr;
  P.wd = nc > 0 ? static_cast<const uint8_t*>(w->wd) : nullptr;
  P.ld_r = w->ld_r * 2;
  P.ld_g = nc > 0 ? w->ld_g * 2 : 0;
  P.ld_u = nc > 0 ? w->ld_u * 2 : 0;
  P.ld_d = nc > 0 ? w->ld_d * 2 : 0;
  P.p_ffn = static_cast<uint16_t*>(io->ffn_partial);
  P.y = static_cast<uint16_t*>(io->y);
  char* base = static_cast<char*>(ws);
  P.sync = reinterpret_cast<unsigned*>(base + L.sync);
  P.logits = reinterpret_cast<float*>(base + L.logits);
  P.m = reinterpret_cast<float*>(base + L.m);
  P.sel_out = sel_out;
  P.prob_out = prob_out;

  const int kmax = std::max(dec::padded(P.H, dec::FMT_F16), top_k * L.npe);
  const size_t lds = sizeof(float) * (kmax / 2 + dec::MAX_SLOTS + 16 + 2 * dec::MOE_MAX_K);
  if (lds > di->max_lds)
    return fail(VT_ERR_UNSUPPORTED, "shape needs %zu bytes of LDS, device has %zu", lds, di->max_lds);
  // every workgroup resident (one per CU): grid barriers separate the phases
  int per_cu = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, dec::moe_kernel, dec::NT, lds);
  if (e != hipSuccess) return fail(VT_ERR_HIP, "occupancy query: %s", hipGetErrorString(e));
  if (per_cu < 1) return fail(VT_ERR_UNSUPPORTED, "MoE kernel does not fit on a CU with %zu bytes of LDS", lds);
  hipLaunchKernelGGL(dec::moe_kernel, dim3(di->cus), dim3(dec::NT), lds, static_cast<hipStream_t>(stream), P);
  e = hipGetLastError();
  if (e != hipSuccess) return fail(VT_ERR_HIP, "MoE launch: %s", hipGetErrorString(e));
  return VT_OK;
}
