// Prefill chunk of one device's shard on gfx950 matrix cores.
//
// Paper Sec. 2.1 (LLM Inference): the prompt's tokens are processed in
// parallel and their K and V are accumulated into the KV cache; with the
// tensor-parallel shard of Sec. 3.2.1 each device does its heads and FFN
// columns. For T tokens at positions pos0..pos0+T-1 the projections are
// dense GEMMs (M = T), run here on fp16 MFMA (v_mfma_f32_32x32x16_f16) with
// fp32 accumulation:
//   rmsnorm_rows   U = fp16(RMSNorm(X) * g_attn)
//   gemm           QKV = U [Wq; Wk; Wv]^T              (fp32 out)
//   rope_append    Q = fp16(RoPE(q) / sqrt(d)); K, V -> cache at pos0+t
//   attn_prefill   O = causal softmax(Q K^T) V, token t sees 0..pos0+t
//   gemm           P_attn = O Wo^T; H = X + P_attn + peer (epilogue)
//   rmsnorm_rows   W = fp16(RMSNorm(H) * g_ffn)
//   gemm           GU = W [Wg; Wu]^T                   (fp32 out)
//   silu_gate      M = fp16(silu(G) * U), zero-padded to the row stride
//   gemm           P_ffn = M Wd^T; Y = H + P_ffn + peer (epilogue)
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <mutex>
#include <vector>

#include "device.hpp"
#include "internal.hpp"

namespace vt {
namespace pf {

typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ f32x16 mfma32(const u32x4 a, const u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

// The GEMMs' activation operands (A) are stored k-step-major: the 16 k
// values of token m in k-step s are halves [(s * M + m) * 16, +16), so the 32
// tokens x 16 k of one MFMA fragment are one contiguous 1 KiB load. K is
// padded with zeros to a multiple of 16.
__device__ __forceinline__ int64_t kmajor(int k, int m, int M) {
  return (static_cast<int64_t>(k >> 4) * M + m) * 16 + (k & 15);
}

// ---------------------------------------------------------------------------
// Split-K GEMM   P[s][m][n] = sum over k-slice s of A[m][k] * B[n][k]
// (fp16 in, fp32 out). M is the chunk's tokens, N the shard's output
// features, K the input features (a multiple of 8). A is k-step-major (see
// kmajor) with zeros past K; B is row-major. The weights (B) are the large
// operand and are streamed once; A is small and re-read from L2 by every N
// tile. The K range is cut into ``splits`` slices so that one launch has
// about one workgroup per compute unit; each slice writes its own fp32 slab
// and the consumer kernel adds the slabs (no atomics, fixed summation order).
//
// Tile 128 tokens x 128 features x 64 k per 256-thread workgroup, two
// workgroups per compute unit (one's barrier and LDS waits are covered by the
// other's MFMAs). Wave w owns tokens 32w..32w+31 and all 128 features as
// 1 x 4 MFMA tiles (32 x 32 x 16 fp16). A wave's A fragments are its own, so they go from global
// memory straight into registers (one contiguous 1 KiB load each, thanks to
// the k-step-major layout), through a ring that runs 8 k-steps (two k-tiles)
// ahead. The B tile is shared by the four waves and is staged in LDS
// (two stages, rows padded by 8 halves; the loads of k-tile i+2 are issued
// before k-tile i is multiplied). Staging only B halves the LDS traffic of
// staging both. Every load is unconditional (out-of-range lanes use an offset
// past the buffer and read zero), so the compiler's wait counts stay exact.
//
// B's rows come from up to three matrices (e.g. Wq, Wk, Wv) placed at
// 8-row-aligned starts of a virtual row space (rows between them read as
// zero). A wave loads 8 consecutive 8-aligned rows per instruction, so each
// load has one source, chosen once per workgroup with scalar selects.
// ---------------------------------------------------------------------------
constexpr int GBM = 128, GBN = 128, GBK = 64, GLD = GBK + 8, GT = 256;
constexpr int KSTEPS = GBK / 16;           // MFMA k-steps per k-tile
constexpr int RING = 2 * KSTEPS;           // A k-steps in flight
constexpr int B_CH = GBN * GBK / 8 / GT;   // 16-byte B chunks per thread per k-tile
constexpr int STAGE = GBN * GLD;           // halves per LDS stage
constexpr int GEMM_LDS_BYTES = 2 * STAGE * 2;
constexpr int GEMM_SLOTS = 512;            // two workgroups per compute unit
constexpr int MAX_SPLITS = 8;

struct BSrc {
  const uint16_t* p;
  int64_t ld;
  int start, rows;  // virtual rows [start, start + rows); start a multiple of 8
};

struct GemmArgs {
  const uint16_t* A;  // k-step-major, ceil(K / 16) k-steps of M tokens
  BSrc b[3];
  int nb;
  float* P;
  int64_t ldp, slab;
  int M, N, K;
  int m_tiles, n_tiles, splits, kps;  // kps: k-tiles per split
};

__global__ void __launch_bounds__(GT, 2) gemm_kernel(GemmArgs g) {
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
  // Workgroups with equal index mod 8 run on one XCD: the M tiles of one
  // (N tile, split) pair get indices that differ by multiples of 8, so their
  // B slice is fetched once into that XCD's L2.
  const int id = blockIdx.x;
  const int slot = id / 8;
  const int unit = (slot / g.m_tiles) * 8 + id % 8;
  const int m_tile = slot % g.m_tiles;
  if (unit >= g.n_tiles * g.splits) return;
  const int n_tile = unit % g.n_tiles, split = unit / g.n_tiles;
  const int m0 = m_tile * GBM, n0 = n_tile * GBN;
  const int t = threadIdx.x, lane = t % kWave;
  const int wave = __builtin_amdgcn_readfirstlane(t / kWave);
  const int KT = (g.K + GBK - 1) / GBK;
  const int kt0 = split * g.kps;
  const int kt_end = min(kt0 + g.kps, KT);
  const int nkt = kt_end - kt0;
  const int ks_end = nkt * KSTEPS;  // k-steps of this split

  rsrc_t rs[3];
#pragma unroll
  for (int j = 0; j < 3; ++j)
    rs[j] = make_rsrc(g.b[j].p, static_cast<uint32_t>(j < g.nb ? g.b[j].rows * g.b[j].ld * 2 : 0));
  const int KS = (g.K + 15) / 16;  // k-steps of A
  const rsrc_t ra = make_rsrc(g.A, static_cast<uint32_t>(KS * g.M * 32));

  // A fragment of this lane: token m, halves 8 (l/32).. of each k-step
  const int am = m0 + wave * 32 + lane % 32;
  const uint32_t aoff = am < g.M ? static_cast<uint32_t>(am * 32 + (lane / 32) * 16) : kOOB;
  const int ks0 = kt0 * KSTEPS;            // the split's first k-step
  // A uniform "out of range" is ORed in as kOOB (valid offsets are below
  // 2^31): a select on a uniform condition would otherwise become a branch,
  // which splits the loop into blocks the scheduler cannot interleave.
  auto load_a = [&](int ks, u32x4& dst) {  // k-step ks of this split
    const int sa = ks0 + ks;
    const uint32_t out = (ks < ks_end && sa < KS) ? 0u : kOOB;
    const uint32_t koff = static_cast<uint32_t>(sa) * static_cast<uint32_t>(g.M) * 32u;
    dst = buf_load16(ra, (aoff + koff) | out | (aoff & kOOB));
  };

  // B chunk offsets (k-independent part); kOOB marks a row past its source
  const int ccol = (t % 8) * 8;
  uint32_t boff[B_CH];
  rsrc_t rsel[B_CH];
#pragma unroll
  for (int u = 0; u < B_CH; ++u) {
    const int r0 = n0 + wave * 8 + u * 32;  // first row of this wave's 8-row group (uniform)
    int j = 2;
    if (r0 < g.b[1].start || g.nb < 2) j = 0;
    else if (r0 < g.b[2].start || g.nb < 3) j = 1;
    const BSrc src = j == 0 ? g.b[0] : (j == 1 ? g.b[1] : g.b[2]);
    rsel[u] = j == 0 ? rs[0] : (j == 1 ? rs[1] : rs[2]);
    const int n = n0 + (t + u * GT) / 8;
    const int r = n - src.start;
    boff[u] = (n < g.N && r >= 0 && r < src.rows) ? static_cast<uint32_t>(r * src.ld * 2) : kOOB;
  }
  auto load_b = [&](int kt, u32x4 (&vb)[B_CH]) {  // k-tile kt (absolute)
    const int k = kt * GBK + ccol;
    const uint32_t out = (kt < kt_end && k < g.K) ? 0u : kOOB;
#pragma unroll
    for (int u = 0; u < B_CH; ++u)
      vb[u] = buf_load16(rsel[u], (boff[u] + static_cast<uint32_t>(k) * 2u) | out | (boff[u] & kOOB));
  };
  auto store_b = [&](uint16_t* st, const u32x4 (&vb)[B_CH]) {
#pragma unroll
    for (int u = 0; u < B_CH; ++u)
      *reinterpret_cast<u32x4*>(st + ((t + u * GT) / 8) * GLD + ccol) = vb[u];
  };

  f32x16 acc[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) acc[b] = f32x16{};

  u32x4 ar[RING];
  // k-tile (from LDS stage st) with A k-steps from ring slots s0..s0+3;
  // each slot is refilled with the k-step RING ahead right after its use.
  // The B fragments of k-step ks+1 are read while k-step ks multiplies.
  auto read_b = [&](const uint16_t* st, int ks, u32x4 (&bf)[4]) {
    const int kc = ks * 16 + 8 * (lane / 32);
#pragma unroll
    for (int b = 0; b < 4; ++b)
      bf[b] = *reinterpret_cast<const u32x4*>(st + (b * 32 + lane % 32) * GLD + kc);
  };
  auto compute = [&](const uint16_t* st, int ks_base, int s0) {
    u32x4 bf[2][4];
    read_b(st, 0, bf[0]);
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      if (ks + 1 < KSTEPS) read_b(st, ks + 1, bf[(ks + 1) & 1]);
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[b] = mfma32(ar[s0 + ks], bf[ks & 1][b], acc[b]);
      load_a(ks_base + ks + RING, ar[s0 + ks]);
    }
  };

  uint16_t* L0 = lds;
  uint16_t* L1 = lds + STAGE;
  u32x4 rb0[B_CH], rb1[B_CH];
#pragma unroll
  for (int s = 0; s < RING; ++s) load_a(s, ar[s]);
  load_b(kt0, rb0);
  load_b(kt0 + 1, rb1);
  store_b(L0, rb0);
  __syncthreads();
  // two k-tiles per trip; an odd count runs one all-zero tile at the end
  // (the scheduling barriers keep the B prefetch ahead of the MFMAs)
  for (int i = 0; i < nkt; i += 2) {
    load_b(kt0 + i + 2, rb0);
    __builtin_amdgcn_sched_barrier(0);
    compute(L0, i * KSTEPS, 0);
    store_b(L1, rb1);
    __syncthreads();
    load_b(kt0 + i + 3, rb1);
    __builtin_amdgcn_sched_barrier(0);
    compute(L1, (i + 1) * KSTEPS, KSTEPS);
    store_b(L0, rb0);
    __syncthreads();
  }

  // accumulator i of tile b: token 8(i/4) + 4(l/32) + i%4, feature l%32
  float* out = g.P + split * g.slab;
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int m = m0 + wave * 32 + 8 * (i / 4) + 4 * (lane / 32) + i % 4;
      const int n = n0 + b * 32 + lane % 32;
      if (m < g.M && n < g.N) out[m * g.ldp + n] = acc[b][i];
    }
}

// Sum over the S split-K slabs of 4 consecutive fp32 values at element i
// (i a multiple of 4); all S loads are issued before the adds.
template <int S>
__device__ __forceinline__ f32x4 slab_sum4(const float* P, int64_t slab, int64_t i) {
  f32x4 v[S];
#pragma unroll
  for (int s = 0; s < S; ++s) v[s] = *reinterpret_cast<const f32x4*>(P + s * slab + i);
#pragma unroll
  for (int s = 1; s < S; ++s) v[0] += v[s];
  return v[0];
}

template <int S>
__device__ __forceinline__ float slab_sum1(const float* P, int64_t slab, int64_t i) {
  float v[S];
#pragma unroll
  for (int s = 0; s < S; ++s) v[s] = P[s * slab + i];
#pragma unroll
  for (int s = 1; s < S; ++s) v[0] += v[s];
  return v[0];
}

// ---------------------------------------------------------------------------
// row-wise helpers
// ---------------------------------------------------------------------------
constexpr int RT = 256;
constexpr int RMAX = 16384 / 8 / RT;  // 16-byte chunks per thread at the largest hidden size

// U[t] = fp16(X[t] / sqrt(mean(X[t]^2) + eps) * g), one workgroup per row
// (grid = the chunk's tokens); U is k-step-major.
__global__ void __launch_bounds__(RT) rmsnorm_rows_kernel(const uint16_t* X, const uint16_t* g,
                                                          uint16_t* U, int H, float eps) {
  __shared__ float red[RT / kWave];
  const int t = blockIdx.x, M = gridDim.x;
  const uint16_t* x = X + static_cast<int64_t>(t) * H;
  float ss = 0.f;
  for (int k8 = threadIdx.x; k8 < H / 8; k8 += RT) {
    float f[8];
    unpack8(load16(x + k8 * 8), f);
#pragma unroll
    for (int e = 0; e < 8; ++e) ss = fmaf(f[e], f[e], ss);
  }
  ss = block_sum<RT>(ss, red);
  const float rstd = 1.0f / sqrtf(ss / static_cast<float>(H) + eps);
  for (int k8 = threadIdx.x; k8 < H / 8; k8 += RT) {
    float f[8], gg[8];
    unpack8(load16(x + k8 * 8), f);
    unpack8(load16(g + k8 * 8), gg);
    uint16_t h[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) h[e] = f2h(f[e] * rstd * gg[e]);
    *reinterpret_cast<u32x4*>(U + kmajor(k8 * 8, t, M)) = pack8(h);
  }
  // zero padding of the last k-step when H is not a multiple of 16
  if ((H & 15) && threadIdx.x == 0)
    *reinterpret_cast<u32x4*>(U + kmajor(H, t, M)) = u32x4{0u, 0u, 0u, 0u};
}

// Residual epilogue of an output projection, one workgroup per token row t:
// p = sum of the slabs, partial[t] = fp16(p), out[t] = fp16(base[t] + p +
// peer[t]) (out may be NULL). With NORM also U[t] = fp16(RMSNorm(out[t]) * g),
// the next sub-layer's normalised input (k-step-major), taken from the
// fp16-rounded row.
template <bool NORM, int S>
__device__ __forceinline__ void resid_body(const float* P, int64_t slab, const uint16_t* base,
                                           const uint16_t* peer, uint16_t* partial, uint16_t* out,
                                           const uint16_t* g, uint16_t* U, int H, float eps) {
  __shared__ float red[RT / kWave];
  const int64_t row = static_cast<int64_t>(blockIdx.x) * H;
  u32x4 hv[RMAX];
  float ss = 0.f;
#pragma unroll
  for (int it = 0; it < RMAX; ++it) {
    const int k8 = threadIdx.x + it * RT;
    if (k8 >= H / 8) break;
    const int64_t i = row + k8 * 8;
    const f32x4 p0 = slab_sum4<S>(P, slab, i), p1 = slab_sum4<S>(P, slab, i + 4);
    const float p[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
    float b[8], pe[8];
    unpack8(load16(base + i), b);
    if (peer) unpack8(load16(peer + i), pe);
    uint16_t ph[8], oh[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      ph[e] = f2h(p[e]);
      oh[e] = f2h(b[e] + p[e] + (peer ? pe[e] : 0.f));
      const float o = h2f(oh[e]);
      ss = fmaf(o, o, ss);
    }
    *reinterpret_cast<u32x4*>(partial + i) = pack8(ph);
    hv[it] = pack8(oh);
    if (out) *reinterpret_cast<u32x4*>(out + i) = hv[it];
  }
  if (!NORM) return;
  ss = block_sum<RT>(ss, red);
  const float rstd = 1.0f / sqrtf(ss / static_cast<float>(H) + eps);
#pragma unroll
  for (int it = 0; it < RMAX; ++it) {
    const int k8 = threadIdx.x + it * RT;
    if (k8 >= H / 8) break;
    float f[8], gg[8];
    unpack8(hv[it], f);
    unpack8(load16(g + k8 * 8), gg);
    uint16_t u[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) u[e] = f2h(f[e] * rstd * gg[e]);
    *reinterpret_cast<u32x4*>(U + kmajor(k8 * 8, blockIdx.x, gridDim.x)) = pack8(u);
  }
  if ((H & 15) && threadIdx.x == 0)
    *reinterpret_cast<u32x4*>(U + kmajor(H, blockIdx.x, gridDim.x)) = u32x4{0u, 0u, 0u, 0u};
}

template <int S>
__global__ void __launch_bounds__(RT) resid_norm_kernel(const float* P, int64_t slab, const uint16_t* base,
                                                        const uint16_t* peer, uint16_t* partial,
                                                        uint16_t* out, const uint16_t* g, uint16_t* U,
                                                        int H, float eps) {
  resid_body<true, S>(P, slab, base, peer, partial, out, g, U, H, eps);
}

template <int S>
__global__ void __launch_bounds__(RT) resid_only_kernel(const float* P, int64_t slab, const uint16_t* base,
                                                        const uint16_t* peer, uint16_t* partial,
                                                        uint16_t* out, const uint16_t* g, uint16_t* U,
                                                        int H, float eps) {
  resid_body<false, S>(P, slab, base, peer, partial, out, g, U, H, eps);
}

// From the raw projections QKV[t] = [q (nq*d) | k (nkv*d) | v (nkv*d)] of
// token t at position pos0 + t (summed over the slabs): Q[t] = fp16(RoPE(q)
// / sqrt(d)); the rotated k and v go to slot pos0 + t of each KV head. One
// workgroup per token.
template <int S>
__global__ void __launch_bounds__(RT) rope_append_kernel(const float* P, int64_t slab, int ldq,
                                                         uint16_t* Q, uint16_t* kc, uint16_t* vc, int nq,
                                                         int nkv, int d, int cap, int pos0, float base) {
  const int t = blockIdx.x;
  const int pos = pos0 + t;
  const int64_t row = static_cast<int64_t>(t) * ldq;
  const float scale = 1.0f / sqrtf(static_cast<float>(d));
  // 4 consecutive values (2 rotary pairs) per step, d / 4 steps per head;
  // RT is a multiple of d / 4, so a thread keeps one column group c4 for all
  // its heads and evaluates its two angles once.
  const int per_head = d / 4;
  const int c4 = (threadIdx.x % per_head) * 4;
  float ca, sa, cb, sb;
  rope_angle(pos, c4 / 2, d, base, ca, sa);
  rope_angle(pos, c4 / 2 + 1, d, base, cb, sb);
  for (int head = threadIdx.x / per_head; head < nq + nkv; head += RT / per_head) {
    const f32x4 v = slab_sum4<S>(P, slab, row + head * d + c4);
    const float r0 = v.x * ca - v.y * sa, r1 = v.x * sa + v.y * ca;
    const float r2 = v.z * cb - v.w * sb, r3 = v.z * sb + v.w * cb;
    uint16_t* o;
    float sc;
    if (head < nq) {
      o = Q + static_cast<int64_t>(t) * nq * d + head * d + c4;
      sc = scale;
    } else {
      o = kc + (static_cast<int64_t>(head - nq) * cap + pos) * d + c4;
      sc = 1.f;
    }
    const unsigned w0 = f2h(r0 * sc) | (static_cast<unsigned>(f2h(r1 * sc)) << 16);
    const unsigned w1 = f2h(r2 * sc) | (static_cast<unsigned>(f2h(r3 * sc)) << 16);
    *reinterpret_cast<uint2*>(o) = make_uint2(w0, w1);
  }
  for (int idx = threadIdx.x; idx < nkv * d / 4; idx += RT) {
    const int g = (idx * 4) / d, dd = idx * 4 - g * d;
    const f32x4 v = slab_sum4<S>(P, slab, row + (nq + nkv) * d + idx * 4);
    const unsigned w0 = f2h(v.x) | (static_cast<unsigned>(f2h(v.y)) << 16);
    const unsigned w1 = f2h(v.z) | (static_cast<unsigned>(f2h(v.w)) << 16);
    *reinterpret_cast<uint2*>(vc + (static_cast<int64_t>(g) * cap + pos) * d + dd) = make_uint2(w0, w1);
  }
}

// Mg[t][j] = fp16(silu(G[t][j]) * Up[t][j]) for j < F, zero for F <= j < kpad
// (k-step-major); G and Up are columns j and up0 + j of the summed slabs (row
// stride ldp). One workgroup per token.
template <int S>
__global__ void __launch_bounds__(RT) silu_gate_kernel(const float* P, int64_t slab, int64_t ldp,
                                                       int up0, uint16_t* Mg, int F, int kpad) {
  const int t = blockIdx.x;
  const int64_t row = static_cast<int64_t>(t) * ldp;
  for (int j = threadIdx.x; j < kpad; j += RT) {
    float m = 0.f;
    if (j < F) {
      const float gt = slab_sum1<S>(P, slab, row + j);
      const float up = slab_sum1<S>(P, slab, row + up0 + j);
      m = gt / (1.0f + __expf(-gt)) * up;
    }
    Mg[kmajor(j, t, gridDim.x)] = f2h(m);
  }
}

// ---------------------------------------------------------------------------
// Causal attention of the chunk (flash-style, MFMA)
//
// One workgroup of AW waves per (query head j, block of 32 queries); wave w
// takes key blocks w, w + AW, ... and keeps its own online softmax (running
// max and sum per query) and output; the AW partial results are merged
// through LDS at the end. Per block of 32 keys a wave computes S^T = K_blk
// Q_blk^T with one 32x32 MFMA tile (K = head_dim), so each lane owns one
// query (column) and 16 of the 32 keys; the partner lane (l ^ 32) owns the
// other 16. The keys are staged into the wave's LDS with rows permuted by
// swapping bits 2 and 3 of the row index: then the 8 accumulators a lane
// feeds into each P.V k-step are exactly the 8 consecutive keys the MFMA
// operand layout asks for, and the probabilities go to the second MFMA
// (O^T += V_blk^T P^T) without any shuffle. V is staged row-major like K
// (16-byte writes) and that MFMA's V^T operand (8 keys of one dimension per
// lane) is gathered with eight 2-byte reads; with rows of D + 8 halves the
// two half-waves of each read fall 32 banks apart. A wave only touches its
// own LDS region inside the loop, so the loop needs no workgroup barrier.
// The output O (the O projection's input) is written k-step-major.
// ---------------------------------------------------------------------------
constexpr int QB = 32, KB = 32, AW = 8;

__device__ __forceinline__ int swap_bits23(int r) {
  return (r & ~0xC) | ((r & 4) << 1) | ((r & 8) >> 1);
}

template <int D>
struct AttnLds {
  static constexpr int KLD = D + 8;   // row stride of the K and V tiles (halves)
  static constexpr int OLD = D + 4;   // row stride of a wave's fp32 output in the merge
  static constexpr int WAVE_HALVES = 2 * KB * KLD;
  static_assert(WAVE_HALVES * 2 >= (QB * OLD + 2 * QB) * 4, "merge buffer must fit a wave's region");
};

template <int D>
__global__ void __launch_bounds__(AW * kWave) attn_prefill_kernel(const uint16_t* Q, uint16_t* O,
                                                                  const uint16_t* kc, const uint16_t* vc,
                                                                  int T, int nq, int G, int cap, int pos0,
                                                                  int window) {
  using LY = AttnLds<D>;
  constexpr int KLD = LY::KLD, OLD = LY::OLD;
  __shared__ __attribute__((aligned(16))) uint16_t smem[AW * LY::WAVE_HALVES];
  const int lane = threadIdx.x % kWave;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  uint16_t* Ks = smem + wave * LY::WAVE_HALVES;
  uint16_t* Vs = Ks + KB * KLD;
  // Workgroups with equal index mod 8 run on one XCD: the query blocks of a
  // head get indices that differ by multiples of 8, so the head's K/V comes
  // from HBM once into that XCD's L2.
  const int nqb = (T + QB - 1) / QB;
  const int j = blockIdx.x % 8 + 8 * (blockIdx.x / (8 * nqb)), qb = (blockIdx.x / 8) % nqb;
  if (j >= nq) return;
  const int g = j / G;
  const int t0 = qb * QB;
  const int tq = t0 + lane % 32;  // this lane's query (token index)
  const int qpos = pos0 + tq;
  constexpr int NKS = D / 16;     // MFMA k-steps over the head dimension

  // Q^T operand: lane supplies Q[tq][16 ks + 8 (l/32) + e]
  u32x4 qf[NKS];
  {
    const int tqc = min(tq, T - 1);
    const uint16_t* qrow = Q + (static_cast<int64_t>(tqc) * nq + j) * D;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) qf[ks] = load16(qrow + ks * 16 + 8 * (lane / 32));
  }
  f32x16 o[D / 32];
#pragma unroll
  for (int mt = 0; mt < D / 32; ++mt) o[mt] = f32x16{};
  float mrun = -INFINITY, lrun = 0.f;

  const int last_key = pos0 + min(t0 + QB, T) - 1;  // largest position any query sees
  const int nkb = last_key / KB + 1;
  // a sliding window: the block's first query sees nothing before this key
  const int kb0 = window > 0 ? max(0, pos0 + t0 - window + 1) / KB : 0;
  const uint16_t* kbase = kc + static_cast<int64_t>(g) * cap * D;
  const uint16_t* vbase = vc + static_cast<int64_t>(g) * cap * D;
  constexpr int CH = KB * D / 8;     // 16-byte chunks per K (or V) tile
  constexpr int CPL = CH / kWave;    // chunks per lane
  // Key block kb's chunks into registers; positions past last_key (never
  // attended) read as zero. Loads are unconditional (clamped position) so
  // the block is fetched in one round trip.
  u32x4 kreg[CPL], vreg[CPL];
  auto fetch = [&](int kb) {
#pragma unroll
    for (int u = 0; u < CPL; ++u) {
      const int c = lane + u * kWave;
      const int key = c / (D / 8), col = (c % (D / 8)) * 8;
      const int p = min(kb * KB + key, last_key);
      kreg[u] = load16(kbase + static_cast<int64_t>(p) * D + col);
      vreg[u] = load16(vbase + static_cast<int64_t>(p) * D + col);
    }
  };
  fetch(min(kb0 + wave, nkb - 1));
  for (int kb = kb0 + wave; kb < nkb; kb += AW) {
    const int p0 = kb * KB;
    // stage K (rows permuted) and V (row-major), then start the next block
#pragma unroll
    for (int u = 0; u < CPL; ++u) {
      const int c = lane + u * kWave;
      const int key = c / (D / 8), col = (c % (D / 8)) * 8;
      const bool live = p0 + key <= last_key;
      const u32x4 kv = live ? kreg[u] : u32x4{0u, 0u, 0u, 0u};
      const u32x4 vv = live ? vreg[u] : u32x4{0u, 0u, 0u, 0u};
      *reinterpret_cast<u32x4*>(Ks + swap_bits23(key) * KLD + col) = kv;
      *reinterpret_cast<u32x4*>(Vs + key * KLD + col) = vv;
    }
    // LDS operations of one wave complete in issue order; this keeps the
    // compiler from moving the tile reads above the writes
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    fetch(min(kb + AW, nkb - 1));
    // S^T (keys x queries)
    f32x16 s = f32x16{};
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const u32x4 kf =
          *reinterpret_cast<const u32x4*>(Ks + (lane % 32) * KLD + ks * 16 + 8 * (lane / 32));
      s = mfma32(kf, qf[ks], s);
    }
    // accumulator i: LDS row 8(i/4) + 4(l/32) + i%4 holds key p0 + swap_bits23(row)
    float bm = -INFINITY;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int key = swap_bits23(8 * (i / 4) + 4 * (lane / 32) + i % 4);
      if (p0 + key > qpos || tq >= T || (window > 0 && p0 + key <= qpos - window)) s[i] = -INFINITY;
      bm = fmaxf(bm, s[i]);
    }
    bm = fmaxf(bm, __shfl_xor(bm, 32, kWave));
    const float mnew = fmaxf(mrun, bm);
    const float alpha = mrun == -INFINITY ? 0.f : __expf(mrun - mnew);
    float ps = 0.f;
    uint16_t ph[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float e = s[i] == -INFINITY ? 0.f : __expf(s[i] - mnew);
      ps += e;
      ph[i] = f2h(e);
    }
    ps += __shfl_xor(ps, 32, kWave);
    lrun = lrun * alpha + ps;
    mrun = mnew;
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
      for (int i = 0; i < 16; ++i) o[mt][i] *= alpha;
    // P^T operand for key step s2: keys 16 s2 + 8 (l/32) + e = accumulators 8 s2 + e
    u32x4 pf[2];
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      pf[s2].x = ph[8 * s2 + 0] | (static_cast<unsigned>(ph[8 * s2 + 1]) << 16);
      pf[s2].y = ph[8 * s2 + 2] | (static_cast<unsigned>(ph[8 * s2 + 3]) << 16);
      pf[s2].z = ph[8 * s2 + 4] | (static_cast<unsigned>(ph[8 * s2 + 5]) << 16);
      pf[s2].w = ph[8 * s2 + 6] | (static_cast<unsigned>(ph[8 * s2 + 7]) << 16);
    }
    // V^T operand for dimension tile mt, key step s2: lane l takes dimension
    // 32 mt + l%32 of keys 16 s2 + 8 (l/32) .. +7
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        const uint16_t* vcol = Vs + (s2 * 16 + 8 * (lane / 32)) * KLD + mt * 32 + lane % 32;
        uint16_t vh[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) vh[e] = vcol[e * KLD];
        o[mt] = mfma32(pack8(vh), pf[s2], o[mt]);
      }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
  }

  // merge the AW partial results: wave w's region holds its output O_w
  // ([query][dim] fp32) and its running max and sum per query
  __syncthreads();
  float* Om = reinterpret_cast<float*>(Ks);
  float* mlw = Om + QB * OLD;
  // O^T accumulator i of tile mt: dim 32 mt + 8(i/4) + 4(l/32) + i%4, query l%32
#pragma unroll
  for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
    for (int i = 0; i < 16; ++i)
      Om[(lane % 32) * OLD + mt * 32 + 8 * (i / 4) + 4 * (lane / 32) + i % 4] = o[mt][i];
  if (lane < 32) {
    mlw[lane] = mrun;
    mlw[QB + lane] = lrun;
  }
  __syncthreads();
  // thread -> (query, 8 consecutive dims)
  constexpr int CPQ = D / 8;  // 8-dim chunks per query
  for (int c = threadIdx.x; c < QB * CPQ; c += AW * kWave) {
    const int q = c / CPQ, d0 = (c % CPQ) * 8;
    if (t0 + q >= T) continue;
    float mw[AW], mstar = -INFINITY;
#pragma unroll
    for (int w = 0; w < AW; ++w) {
      const float* mlv = reinterpret_cast<const float*>(smem + w * LY::WAVE_HALVES) + QB * OLD;
      mw[w] = mlv[q];
      mstar = fmaxf(mstar, mw[w]);
    }
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f}, l = 0.f;
#pragma unroll
    for (int w = 0; w < AW; ++w) {
      const float* ow = reinterpret_cast<const float*>(smem + w * LY::WAVE_HALVES);
      const float sc = mw[w] == -INFINITY ? 0.f : __expf(mw[w] - mstar);
      l += sc * ow[QB * OLD + QB + q];
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += sc * ow[q * OLD + d0 + e];
    }
    const float inv = 1.0f / l;
    uint16_t h[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) h[e] = f2h(acc[e] * inv);
    *reinterpret_cast<u32x4*>(O + kmajor(j * D + d0, t0 + q, T)) = pack8(h);
  }
}

}  // namespace pf

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
namespace {

// Split-K choice of a GEMM: enough slices of whole k-tiles for about two
// rounds of resident workgroups (GEMM_SLOTS each), at most 4. Measured on the
// 256-token chunk of the 7B 50% shard: 4 slices beat 2, 3, 6 and 8 for the
// gate/up, O and down GEMMs and are within 4% of 5 for QKV; more slices add
// fp32 slab traffic, fewer leave compute units idle.
struct Split {
  int m_tiles, n_tiles, splits, kps;
};

Split choose_split(int M, int N, int K) {
  Split s;
  s.m_tiles = (M + pf::GBM - 1) / pf::GBM;
  s.n_tiles = (N + pf::GBN - 1) / pf::GBN;
  const int KT = std::max(1, (K + pf::GBK - 1) / pf::GBK);
  const int tiles = std::max(1, s.m_tiles * s.n_tiles);
  const int want = std::max(1, std::min({KT, 4, (2 * pf::GEMM_SLOTS + tiles - 1) / tiles}));
  s.kps = (KT + want - 1) / want;
  s.splits = (KT + s.kps - 1) / s.kps;
  return s;
}

// The shard's prefill GEMMs for T tokens: QKV, O, gate/up, down. N counts
// virtual rows of B (the up rows start at the 8-aligned row after the gate
// rows); K is rounded up to a multiple of 8 (the padding multiplies zeros).
struct PrefillGemms {
  int M, N[4], K[4], up0;
};

PrefillGemms prefill_gemms(const vt_shard_spec& s, int32_t T) {
  const vt_shard_info& in = s.info;
  const int H = s.dims.hidden, d = s.dims.head_dim;
  PrefillGemms g;
  g.M = T;
  g.N[0] = (in.n_q_heads + 2 * in.n_kv_heads) * d;
  g.K[0] = H;
  g.N[1] = H;
  g.K[1] = in.n_q_heads * d;
  g.up0 = (in.n_cols + 7) / 8 * 8;
  g.N[2] = g.up0 + in.n_cols;
  g.K[2] = H;
  g.N[3] = H;
  g.K[3] = std::max(8, g.up0);
  return g;
}

struct PrefillWs {
  size_t u, q, o, m, part, total;
};

inline int64_t rup(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

PrefillWs prefill_layout(const vt_shard_spec& s, int32_t T) {
  const vt_shard_info& in = s.info;
  const int64_t H = s.dims.hidden, d = s.dims.head_dim;
  const PrefillGemms gm = prefill_gemms(s, T);
  int64_t part = 0;  // one region serves the four GEMMs' slabs in turn
  for (int i = 0; i < 4; ++i) {
    const Split sp = choose_split(gm.M, gm.N[i], gm.K[i]);
    part = std::max<int64_t>(part, static_cast<int64_t>(sp.splits) * T * gm.N[i] * 4);
  }
  PrefillWs w{};
  size_t off = workspace_sync_bytes(s);  // leave the decode synchronisation words alone
  auto take = [&](int64_t bytes) {
    size_t at = off;
    off += static_cast<size_t>(rup(std::max<int64_t>(bytes, 16), 256));
    return at;
  };
  // k-step-major activation operands, K padded to a multiple of 16
  w.u = take(2 * T * rup(H, 16));
  w.q = take(2 * T * in.n_q_heads * d);
  w.o = take(2 * T * std::max<int64_t>(rup(in.n_q_heads * d, 16), 16));
  w.m = take(2 * T * std::max<int64_t>(rup(in.n_cols, 16), 16));
  w.part = take(part);
  w.total = off;
  return w;
}

// Launches P = A B^T as split-K slabs; returns the slab count via *splits.
vt_status launch_gemm(pf::GemmArgs a, float* P, hipStream_t s, int* splits) {
  {
    // the GEMM's dynamic LDS exceeds the default limit: raise it once per device
    static std::mutex mu;
    static std::vector<char> done;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(VT_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    std::lock_guard<std::mutex> lk(mu);
    if (static_cast<int>(done.size()) <= dev) done.resize(dev + 1, 0);
    if (!done[dev]) {
      e = hipFuncSetAttribute(reinterpret_cast<const void*>(pf::gemm_kernel),
                              hipFuncAttributeMaxDynamicSharedMemorySize, pf::GEMM_LDS_BYTES);
      if (e != hipSuccess)
        return fail(VT_ERR_HIP, "gemm LDS attribute: %s", hipGetErrorString(e));
      done[dev] = 1;
    }
  }
  const Split sp = choose_split(a.M, a.N, a.K);
  a.m_tiles = sp.m_tiles;
  a.n_tiles = sp.n_tiles;
  a.splits = sp.splits;
  a.kps = sp.kps;
  a.P = P;
  a.ldp = a.N;
  a.slab = static_cast<int64_t>(a.M) * a.N;
  *splits = sp.splits;
  if (a.M == 0 || a.N == 0) return VT_OK;
  const int units = sp.n_tiles * sp.splits;
  const int groups = (units + 7) / 8;
  hipLaunchKernelGGL(pf::gemm_kernel, dim3(groups * 8 * sp.m_tiles), dim3(pf::GT),
                     pf::GEMM_LDS_BYTES, s, a);
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? VT_OK : fail(VT_ERR_HIP, "gemm launch: %s", hipGetErrorString(e));
}

pf::BSrc bsrc(const void* p, int64_t ld, int start, int rows) {
  return pf::BSrc{static_cast<const uint16_t*>(p), ld, start, rows};
}

// Launch helper for kernels templated on the split-K slab count.
#define VT_SPLIT_DISPATCH(KERNEL, ...)                                           \
  switch (splits) {                                                              \
    case 1: hipLaunchKernelGGL(KERNEL<1>, __VA_ARGS__); break;                   \
    case 2: hipLaunchKernelGGL(KERNEL<2>, __VA_ARGS__); break;                   \
    case 3: hipLaunchKernelGGL(KERNEL<3>, __VA_ARGS__); break;                   \
    case 4: hipLaunchKernelGGL(KERNEL<4>, __VA_ARGS__); break;                   \
    case 5: hipLaunchKernelGGL(KERNEL<5>, __VA_ARGS__); break;                   \
    case 6: hipLaunchKernelGGL(KERNEL<6>, __VA_ARGS__); break;                   \
    case 7: hipLaunchKernelGGL(KERNEL<7>, __VA_ARGS__); break;                   \
    default: hipLaunchKernelGGL(KERNEL<8>, __VA_ARGS__); break;                  \
  }

}  // namespace

size_t prefill_workspace_bytes(const vt_shard_spec& s, int32_t max_tokens, int32_t) {
  return prefill_layout(s, max_tokens).total;
}

}  // namespace vt

using namespace vt;

extern "C" vt_status vt_layer_prefill_chunk(const vt_shard_spec* spec, const vt_layer_weights* w,
                                            vt_kv_view* kv, const vt_layer_io* io, int32_t n_tok,
                                            int32_t pos0, uint32_t phases, void* ws, size_t ws_bytes,
                                            void* stream) {
  clear_error();
  if (!spec || !io) return fail(VT_ERR_ARG, "null spec or io");
  if (phases & ~(VT_ATTN | VT_FFN)) return fail(VT_ERR_ARG, "unknown phase bits 0x%x", phases);
  const bool attn = phases & VT_ATTN, ffn = phases & VT_FFN;
  if (!attn && !ffn) return fail(VT_ERR_ARG, "no phase selected");
  if (n_tok < 1 || n_tok > 65536) return fail(VT_ERR_ARG, "n_tok %d outside 1..65536", n_tok);
  const vt_layer_dims& D = spec->dims;
  const vt_shard_info& in = spec->info;
  vt_status st = check_weights(*spec, w, attn, ffn);
  if (st != VT_OK) return st;
  auto vec = [&](const void* p, const char* name, bool required) -> vt_status {
    if (!p) return required ? fail(VT_ERR_ARG, "%s is NULL", name) : VT_OK;
    if (!aligned16(p)) return fail(VT_ERR_ALIGN, "%s is not 16-byte aligned", name);
    return VT_OK;
  };
  if (attn) {
    if ((st = check_kv(*spec, kv, pos0, n_tok)) != VT_OK) return st;
    if ((st = vec(io->x, "x", true)) != VT_OK) return st;
    if ((st = vec(io->peer_attn, "peer_attn", false)) != VT_OK) return st;
    if ((st = vec(io->attn_partial, "attn_partial", true)) != VT_OK) return st;
  }
  if ((st = vec(io->h, "h", true)) != VT_OK) return st;
  if (ffn) {
    if ((st = vec(io->peer_ffn, "peer_ffn", false)) != VT_OK) return st;
    if ((st = vec(io->ffn_partial, "ffn_partial", true)) != VT_OK) return st;
    if ((st = vec(io->y, "y", false)) != VT_OK) return st;
  }
  const int64_t H = D.hidden, d = D.head_dim;
  if (attn && in.n_q_heads == 0)
    return fail(VT_ERR_UNSUPPORTED, "prefill of a shard without heads");
  if (ffn && in.n_cols == 0)
    return fail(VT_ERR_UNSUPPORTED, "prefill of a shard without FFN columns");
  // activation operands of the GEMMs are read through 2 GiB buffer ranges
  if (static_cast<int64_t>(n_tok) * std::max<int64_t>({H + 16, in.n_q_heads * d, in.n_cols + 16}) * 2 >=
      kMaxBufferBytes)
    return fail(VT_ERR_UNSUPPORTED, "chunk of %d tokens too large for 2 GiB activation buffers", n_tok);
  const PrefillWs L = prefill_layout(*spec, n_tok);
  if (!ws || ws_bytes < L.total)
    return fail(VT_ERR_WORKSPACE, "workspace %zu bytes, need %zu", ws_bytes, L.total);
  if (!aligned16(ws)) return fail(VT_ERR_ALIGN, "workspace not 16-byte aligned");

  char* base = static_cast<char*>(ws);
  uint16_t* U = reinterpret_cast<uint16_t*>(base + L.u);
  uint16_t* Qr = reinterpret_cast<uint16_t*>(base + L.q);
  uint16_t* Ob = reinterpret_cast<uint16_t*>(base + L.o);
  uint16_t* Mb = reinterpret_cast<uint16_t*>(base + L.m);
  float* P = reinterpret_cast<float*>(base + L.part);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int nq = in.n_q_heads, nkv = in.n_kv_heads, F = in.n_cols;
  const int G = D.n_heads / D.n_kv_heads;
  const int kpad_f = std::max(16, (F + 15) / 16 * 16);  // k-step-major width of the SiLU-gate output
  const PrefillGemms gm = prefill_gemms(*spec, n_tok);
  int splits = 1;
  auto check = [&](const char* what) -> vt_status {
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? VT_OK : fail(VT_ERR_HIP, "%s launch: %s", what, hipGetErrorString(e));
  };
  auto slab = [&](int i) { return static_cast<int64_t>(n_tok) * gm.N[i]; };

  if (attn) {
    hipLaunchKernelGGL(pf::rmsnorm_rows_kernel, dim3(n_tok), dim3(pf::RT), 0, s,
                       static_cast<const uint16_t*>(io->x), static_cast<const uint16_t*>(w->g_attn), U,
                       static_cast<int>(H), D.rms_eps);
    if ((st = check("rmsnorm")) != VT_OK) return st;
    pf::GemmArgs a{};
    a.A = U;
    a.K = gm.K[0];
    a.M = n_tok;
    a.N = gm.N[0];
    const int qd = nq * static_cast<int>(d), kd = nkv * static_cast<int>(d);
    a.b[0] = bsrc(w->wq, w->ld_q, 0, qd);
    a.b[1] = bsrc(w->wk, w->ld_k, qd, kd);
    a.b[2] = bsrc(w->wv, w->ld_v, qd + kd, kd);
    a.nb = 3;
    if ((st = launch_gemm(a, P, s, &splits)) != VT_OK) return st;
    VT_SPLIT_DISPATCH(pf::rope_append_kernel, dim3(n_tok), dim3(pf::RT), 0, s, P, slab(0), gm.N[0], Qr,
                      static_cast<uint16_t*>(kv->k), static_cast<uint16_t*>(kv->v), nq, nkv,
                      static_cast<int>(d), kv->capacity, pos0, D.rope_base);
    if ((st = check("rope_append")) != VT_OK) return st;
    const int blocks = (nq + 7) / 8 * 8 * ((n_tok + pf::QB - 1) / pf::QB);
    if (d == 128)
      hipLaunchKernelGGL(pf::attn_prefill_kernel<128>, dim3(blocks), dim3(pf::AW * kWave), 0, s, Qr, Ob,
                         static_cast<const uint16_t*>(kv->k), static_cast<const uint16_t*>(kv->v),
                         n_tok, nq, G, kv->capacity, pos0, D.window);
    else
      hipLaunchKernelGGL(pf::attn_prefill_kernel<64>, dim3(blocks), dim3(pf::AW * kWave), 0, s, Qr, Ob,
                         static_cast<const uint16_t*>(kv->k), static_cast<const uint16_t*>(kv->v),
                         n_tok, nq, G, kv->capacity, pos0, D.window);
    if ((st = check("attention")) != VT_OK) return st;
    pf::GemmArgs o{};
    o.A = Ob;
    o.K = gm.K[1];
    o.M = n_tok;
    o.N = gm.N[1];
    o.b[0] = bsrc(w->wo, w->ld_o, 0, gm.N[1]);
    o.nb = 1;
    if ((st = launch_gemm(o, P, s, &splits)) != VT_OK) return st;
    // h = x + p_attn + peer; with FFN to follow also U = RMSNorm(h) * g_ffn
    if (ffn) {
      VT_SPLIT_DISPATCH(pf::resid_norm_kernel, dim3(n_tok), dim3(pf::RT), 0, s, P, slab(1),
                        static_cast<const uint16_t*>(io->x), static_cast<const uint16_t*>(io->peer_attn),
                        static_cast<uint16_t*>(io->attn_partial), static_cast<uint16_t*>(io->h),
                        static_cast<const uint16_t*>(w->g_ffn), U, static_cast<int>(H), D.rms_eps);
    } else {
      VT_SPLIT_DISPATCH(pf::resid_only_kernel, dim3(n_tok), dim3(pf::RT), 0, s, P, slab(1),
                        static_cast<const uint16_t*>(io->x), static_cast<const uint16_t*>(io->peer_attn),
                        static_cast<uint16_t*>(io->attn_partial), static_cast<uint16_t*>(io->h),
                        static_cast<const uint16_t*>(nullptr), static_cast<uint16_t*>(nullptr),
                        static_cast<int>(H), D.rms_eps);
    }
    if ((st = check("attention residual")) != VT_OK) return st;
  }
  if (ffn) {
    if (!attn) {
      hipLaunchKernelGGL(pf::rmsnorm_rows_kernel, dim3(n_tok), dim3(pf::RT), 0, s,
                         static_cast<const uint16_t*>(io->h), static_cast<const uint16_t*>(w->g_ffn),
                         U, static_cast<int>(H), D.rms_eps);
      if ((st = check("rmsnorm")) != VT_OK) return st;
    }
    pf::GemmArgs a{};
    a.A = U;
    a.K = gm.K[2];
    a.M = n_tok;
    a.N = gm.N[2];
    a.b[0] = bsrc(w->wg, w->ld_g, 0, F);
    a.b[1] = bsrc(w->wu, w->ld_u, gm.up0, F);
    a.nb = 2;
    if ((st = launch_gemm(a, P, s, &splits)) != VT_OK) return st;
    VT_SPLIT_DISPATCH(pf::silu_gate_kernel, dim3(n_tok), dim3(pf::RT), 0, s, P, slab(2),
                      static_cast<int64_t>(gm.N[2]), gm.up0, Mb, F, kpad_f);
    if ((st = check("silu_gate")) != VT_OK) return st;
    pf::GemmArgs b{};
    b.A = Mb;
    b.K = gm.K[3];
    b.M = n_tok;
    b.N = gm.N[3];
    b.b[0] = bsrc(w->wd, w->ld_d, 0, gm.N[3]);
    b.nb = 1;
    if ((st = launch_gemm(b, P, s, &splits)) != VT_OK) return st;
    VT_SPLIT_DISPATCH(pf::resid_only_kernel, dim3(n_tok), dim3(pf::RT), 0, s, P, slab(3),
                      static_cast<const uint16_t*>(io->h), static_cast<const uint16_t*>(io->peer_ffn),
                      static_cast<uint16_t*>(io->ffn_partial), static_cast<uint16_t*>(io->y),
                      static_cast<const uint16_t*>(nullptr), static_cast<uint16_t*>(nullptr),
                      static_cast<int>(H), D.rms_eps);
    if ((st = check("ffn residual")) != VT_OK) return st;
  }
  if (attn) kv->len = pos0 + n_tok;
  return VT_OK;
}
