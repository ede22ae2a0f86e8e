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

#include "device.hpp"
#include "internal.hpp"

namespace vt {
namespace pf {

typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ f32x16 mfma32(const u32x4 a, const u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

// Zero the fp16 values at columns >= K of an 8-column chunk starting at col.
__device__ __forceinline__ u32x4 mask_cols(u32x4 w, int col, int K) {
  const int v = K - col;
  if (v >= 8) return w;
  if (v <= 0) return u32x4{0u, 0u, 0u, 0u};
  w.x = v >= 2 ? w.x : (w.x & 0xFFFFu);
  w.y = v >= 4 ? w.y : (v >= 3 ? (w.y & 0xFFFFu) : 0u);
  w.z = v >= 6 ? w.z : (v >= 5 ? (w.z & 0xFFFFu) : 0u);
  w.w = v >= 7 ? (w.w & 0xFFFFu) : 0u;
  return w;
}

// ---------------------------------------------------------------------------
// GEMM  C[M][N] = A[M][K] . B[N][K]^T  (fp16 in, fp32 accumulate)
// B's rows come from two matrices: rows < n1 from B1, the rest from B2.
// Tile 128 x 128 x 32 per 256-thread workgroup; each of the four waves owns a
// 64 x 64 quarter as 2 x 2 MFMA tiles. A and B tiles pass through LDS (rows
// padded by 8 halves); the next k-tile is loaded into registers while the
// current one is multiplied.
// ---------------------------------------------------------------------------
constexpr int BM = 128, BN = 128, BK = 32, LDK = BK + 8, GT = 256;

struct GemmArgs {
  const uint16_t* A;
  int64_t lda;
  const uint16_t* B1;
  int64_t ldb1;
  int n1;
  const uint16_t* B2;
  int64_t ldb2;
  int M, N, K;
  int m_tiles, n_tiles;
};

template <class Epi>
__global__ void __launch_bounds__(GT) gemm_kernel(GemmArgs g, Epi epi) {
  __shared__ __attribute__((aligned(16))) uint16_t As[BM * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[BN * LDK];
  // Workgroups with equal index mod 8 run on one XCD: give the M tiles of an
  // N tile indices that differ by multiples of 8, so B is fetched once into
  // that XCD's L2.
  const int id = blockIdx.x;
  const int slot = id / 8;
  const int n_tile = (slot / g.m_tiles) * 8 + id % 8;
  const int m_tile = slot % g.m_tiles;
  if (n_tile >= g.n_tiles) return;
  const int m0 = m_tile * BM, n0 = n_tile * BN;
  const int t = threadIdx.x, lane = t % kWave, wave = t / kWave;
  const int wm = wave / 2, wn = wave % 2;

  const rsrc_t ra = make_rsrc(g.A, static_cast<uint32_t>(g.M * g.lda * 2));
  const rsrc_t rb1 = make_rsrc(g.B1, static_cast<uint32_t>(g.n1 * g.ldb1 * 2));
  const rsrc_t rb2 =
      make_rsrc(g.B2, static_cast<uint32_t>(static_cast<int64_t>(g.N - g.n1) * g.ldb2 * 2));
  // This thread's two 16-byte chunks of each tile: row id/4, column (id%4)*8.
  int arow[2], brow[2], ccol[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int cid = t + u * GT;
    arow[u] = cid / 4;
    brow[u] = cid / 4;
    ccol[u] = (cid % 4) * 8;
  }
  auto load_a = [&](int k0, int u) -> u32x4 {
    const int m = m0 + arow[u], k = k0 + ccol[u];
    const bool ok = m < g.M && k < g.K;
    const uint32_t off = ok ? static_cast<uint32_t>((m * g.lda + k) * 2) : kOOB;
    return mask_cols(buf_load16(ra, off), k, g.K);
  };
  auto load_b = [&](int k0, int u) -> u32x4 {
    const int n = n0 + brow[u], k = k0 + ccol[u];
    const bool ok = n < g.N && k < g.K;
    const bool first = n < g.n1;
    const int64_t row = first ? n : n - g.n1;
    const int64_t ld = first ? g.ldb1 : g.ldb2;
    const uint32_t off = ok ? static_cast<uint32_t>((row * ld + k) * 2) : kOOB;
    const u32x4 v = first ? buf_load16(rb1, off) : buf_load16(rb2, off);
    return mask_cols(v, k, g.K);
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x16{};

  u32x4 ra_n[2], rb_n[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    ra_n[u] = load_a(0, u);
    rb_n[u] = load_b(0, u);
  }
  for (int k0 = 0; k0 < g.K; k0 += BK) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      *reinterpret_cast<u32x4*>(As + arow[u] * LDK + ccol[u]) = ra_n[u];
      *reinterpret_cast<u32x4*>(Bs + brow[u] * LDK + ccol[u]) = rb_n[u];
    }
    __syncthreads();
    if (k0 + BK < g.K) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        ra_n[u] = load_a(k0 + BK, u);
        rb_n[u] = load_b(k0 + BK, u);
      }
    }
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      u32x4 af[2], bf[2];
#pragma unroll
      for (int a = 0; a < 2; ++a)
        af[a] = *reinterpret_cast<const u32x4*>(As + (wm * 64 + a * 32 + lane % 32) * LDK + ks * 16 +
                                                8 * (lane / 32));
#pragma unroll
      for (int b = 0; b < 2; ++b)
        bf[b] = *reinterpret_cast<const u32x4*>(Bs + (wn * 64 + b * 32 + lane % 32) * LDK + ks * 16 +
                                                8 * (lane / 32));
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) acc[a][b] = mfma32(af[a], bf[b], acc[a][b]);
    }
    __syncthreads();
  }
  // accumulator i of lane l holds row 8(i/4) + 4(l/32) + i%4, column l%32
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int m = m0 + wm * 64 + a * 32 + 8 * (i / 4) + 4 * (lane / 32) + i % 4;
        const int n = n0 + wn * 64 + b * 32 + lane % 32;
        if (m < g.M && n < g.N) epi(m, n, acc[a][b][i]);
      }
}

struct EpiStoreF32 {  // C -> fp32 matrix with row stride ld
  float* c;
  int64_t ld;
  __device__ void operator()(int m, int n, float v) const { c[m * ld + n] = v; }
};

struct EpiResidual {  // partial -> fp16; out = base + partial + peer (fp16)
  uint16_t* partial;
  uint16_t* out;
  const uint16_t* base;
  const uint16_t* peer;
  int64_t ld;
  __device__ void operator()(int m, int n, float v) const {
    const int64_t i = m * ld + n;
    partial[i] = f2h(v);
    if (out) out[i] = f2h(h2f(base[i]) + v + (peer ? h2f(peer[i]) : 0.f));
  }
};

// ---------------------------------------------------------------------------
// row-wise helpers
// ---------------------------------------------------------------------------
constexpr int RT = 256;

// U[t] = fp16(X[t] / sqrt(mean(X[t]^2) + eps) * g), one workgroup per row.
__global__ void __launch_bounds__(RT) rmsnorm_rows_kernel(const uint16_t* X, const uint16_t* g,
                                                          uint16_t* U, int H, float eps) {
  __shared__ float red[RT / kWave];
  const uint16_t* x = X + static_cast<int64_t>(blockIdx.x) * H;
  uint16_t* u = U + static_cast<int64_t>(blockIdx.x) * H;
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
    u32x4 o;
    uint16_t h[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) h[e] = f2h(f[e] * rstd * gg[e]);
    o.x = h[0] | (static_cast<unsigned>(h[1]) << 16);
    o.y = h[2] | (static_cast<unsigned>(h[3]) << 16);
    o.z = h[4] | (static_cast<unsigned>(h[5]) << 16);
    o.w = h[6] | (static_cast<unsigned>(h[7]) << 16);
    *reinterpret_cast<u32x4*>(u + k8 * 8) = o;
  }
}

// From the raw projections QKV[t] = [q (nq*d) | k (nkv*d) | v (nkv*d)] of
// token t at position pos0 + t: Q[t] = fp16(RoPE(q) / sqrt(d)); the rotated
// k and v go to slot pos0 + t of each KV head. One workgroup per token.
__global__ void __launch_bounds__(RT) rope_append_kernel(const float* QKV, int ldq, uint16_t* Q,
                                                         uint16_t* kc, uint16_t* vc, int nq, int nkv,
                                                         int d, int cap, int pos0, float base) {
  const int t = blockIdx.x;
  const int pos = pos0 + t;
  const float* row = QKV + static_cast<int64_t>(t) * ldq;
  const float scale = 1.0f / sqrtf(static_cast<float>(d));
  const int half = d / 2;
  for (int idx = threadIdx.x; idx < (nq + nkv) * half; idx += RT) {
    const int head = idx / half, i = idx - head * half;
    float c0, s0;
    rope_angle(pos, i, d, base, c0, s0);
    const float a = row[head * d + 2 * i], b = row[head * d + 2 * i + 1];
    const float r0 = a * c0 - b * s0, r1 = a * s0 + b * c0;
    if (head < nq) {
      uint16_t* qo = Q + static_cast<int64_t>(t) * nq * d + head * d;
      qo[2 * i] = f2h(r0 * scale);
      qo[2 * i + 1] = f2h(r1 * scale);
    } else {
      const int g = head - nq;
      uint16_t* ko = kc + (static_cast<int64_t>(g) * cap + pos) * d;
      ko[2 * i] = f2h(r0);
      ko[2 * i + 1] = f2h(r1);
    }
  }
  for (int idx = threadIdx.x; idx < nkv * d; idx += RT) {
    const int g = idx / d, dd = idx - g * d;
    vc[(static_cast<int64_t>(g) * cap + pos) * d + dd] = f2h(row[(nq + nkv) * d + idx]);
  }
}

// M[t][j] = fp16(silu(G[t][j]) * Up[t][j]) for j < F, zero for F <= j < ldm.
__global__ void __launch_bounds__(RT) silu_gate_kernel(const float* GU, int ldgu, uint16_t* M, int F,
                                                       int ldm) {
  const int t = blockIdx.x;
  const float* row = GU + static_cast<int64_t>(t) * ldgu;
  for (int j = threadIdx.x; j < ldm; j += RT) {
    float m = 0.f;
    if (j < F) {
      const float gt = row[j], up = row[F + j];
      m = gt / (1.0f + __expf(-gt)) * up;
    }
    M[static_cast<int64_t>(t) * ldm + j] = f2h(m);
  }
}

// ---------------------------------------------------------------------------
// Causal attention of the chunk (flash-style, MFMA)
//
// One wave per (query head j, block of 32 queries). Per block of 32 keys it
// computes S^T = K_blk Q_blk^T with one 32x32 MFMA tile (K = head_dim), so
// each lane owns one query (column) and 16 of the 32 keys; the partner lane
// (l ^ 32) owns the other 16. The keys are staged into LDS with rows
// permuted by swapping bits 2 and 3 of the row index: then the 8
// accumulators a lane feeds into each P.V k-step are exactly the 8
// consecutive keys the MFMA operand layout asks for, and the probabilities
// go to the second MFMA (O^T += V_blk^T P^T) without any shuffle. V is
// staged transposed ([dim][key]) for that MFMA's other operand. Softmax is
// online across key blocks (running max and sum per query).
// ---------------------------------------------------------------------------
constexpr int QB = 32, KB = 32;

__device__ __forceinline__ int swap_bits23(int r) {
  return (r & ~0xC) | ((r & 4) << 1) | ((r & 8) >> 1);
}

template <int D>
__global__ void __launch_bounds__(kWave) attn_prefill_kernel(const uint16_t* Q, uint16_t* O,
                                                             const uint16_t* kc, const uint16_t* vc,
                                                             int T, int nq, int G, int cap, int pos0) {
  constexpr int KLD = D + 8;   // LDS row stride of the K tile (halves)
  constexpr int VLD = KB + 8;  // LDS row stride of the transposed V tile
  __shared__ __attribute__((aligned(16))) uint16_t Ks[KB * KLD];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[D * VLD];
  const int lane = threadIdx.x;
  const int nqb = (T + QB - 1) / QB;
  const int j = blockIdx.x / nqb, qb = blockIdx.x % nqb;
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
  fetch(0);
  for (int kb = 0; kb < nkb; ++kb) {
    const int p0 = kb * KB;
    // stage K (rows permuted) and V (transposed), then start the next block
#pragma unroll
    for (int u = 0; u < CPL; ++u) {
      const int c = lane + u * kWave;
      const int key = c / (D / 8), col = (c % (D / 8)) * 8;
      const bool live = p0 + key <= last_key;
      const u32x4 kv = live ? kreg[u] : u32x4{0u, 0u, 0u, 0u};
      const u32x4 vv = live ? vreg[u] : u32x4{0u, 0u, 0u, 0u};
      *reinterpret_cast<u32x4*>(Ks + swap_bits23(key) * KLD + col) = kv;
      const uint16_t vh[8] = {
          static_cast<uint16_t>(vv.x), static_cast<uint16_t>(vv.x >> 16),
          static_cast<uint16_t>(vv.y), static_cast<uint16_t>(vv.y >> 16),
          static_cast<uint16_t>(vv.z), static_cast<uint16_t>(vv.z >> 16),
          static_cast<uint16_t>(vv.w), static_cast<uint16_t>(vv.w >> 16)};
#pragma unroll
      for (int e = 0; e < 8; ++e) Vt[(col + e) * VLD + key] = vh[e];
    }
    __syncthreads();
    if (kb + 1 < nkb) fetch(kb + 1);
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
      if (p0 + key > qpos || tq >= T) s[i] = -INFINITY;
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
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        const u32x4 vf = *reinterpret_cast<const u32x4*>(Vt + (mt * 32 + lane % 32) * VLD + s2 * 16 +
                                                         8 * (lane / 32));
        o[mt] = mfma32(vf, pf[s2], o[mt]);
      }
    __syncthreads();
  }
  // O^T accumulator i of tile mt: dim 32 mt + 8(i/4) + 4(l/32) + i%4, query l%32
  if (tq < T) {
    const float inv = 1.0f / lrun;
    uint16_t* orow = O + (static_cast<int64_t>(tq) * nq + j) * D;
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
      for (int i = 0; i < 16; ++i) orow[mt * 32 + 8 * (i / 4) + 4 * (lane / 32) + i % 4] = f2h(o[mt][i] * inv);
  }
}

}  // namespace pf

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
namespace {

struct PrefillWs {
  size_t u, qkv, q, o, gu, m, total;
};

inline int64_t rup(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

PrefillWs prefill_layout(const vt_shard_spec& s, int32_t T) {
  const vt_shard_info& in = s.info;
  const int64_t H = s.dims.hidden, d = s.dims.head_dim;
  const int64_t r0 = (in.n_q_heads + 2 * in.n_kv_heads) * d;
  const int64_t fpad = std::max<int64_t>(8, rup(in.n_cols, 8));
  PrefillWs w{};
  size_t off = workspace_sync_bytes(s);  // leave the decode synchronisation words alone
  auto take = [&](int64_t bytes) {
    size_t at = off;
    off += static_cast<size_t>(rup(std::max<int64_t>(bytes, 16), 256));
    return at;
  };
  w.u = take(2 * T * H);
  w.qkv = take(4 * T * r0);
  w.q = take(2 * T * in.n_q_heads * d);
  w.o = take(2 * T * std::max<int64_t>(in.n_q_heads * d, 8));
  w.gu = take(4 * T * 2 * in.n_cols);
  w.m = take(2 * T * fpad);
  w.total = off;
  return w;
}

template <class Epi>
vt_status launch_gemm(const pf::GemmArgs& a0, Epi epi, hipStream_t s) {
  pf::GemmArgs a = a0;
  a.m_tiles = (a.M + pf::BM - 1) / pf::BM;
  a.n_tiles = (a.N + pf::BN - 1) / pf::BN;
  if (a.M == 0 || a.N == 0) return VT_OK;
  const int groups = (a.n_tiles + 7) / 8;
  hipLaunchKernelGGL(pf::gemm_kernel<Epi>, dim3(groups * 8 * a.m_tiles), dim3(pf::GT), 0, s, a, epi);
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? VT_OK : fail(VT_ERR_HIP, "gemm launch: %s", hipGetErrorString(e));
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
  if (static_cast<int64_t>(n_tok) * std::max<int64_t>(H, 2 * in.n_cols + 8) * 4 >= kMaxBufferBytes)
    return fail(VT_ERR_UNSUPPORTED, "chunk of %d tokens too large for 2 GiB activation buffers", n_tok);
  const PrefillWs L = prefill_layout(*spec, n_tok);
  if (!ws || ws_bytes < L.total)
    return fail(VT_ERR_WORKSPACE, "workspace %zu bytes, need %zu", ws_bytes, L.total);
  if (!aligned16(ws)) return fail(VT_ERR_ALIGN, "workspace not 16-byte aligned");

  char* base = static_cast<char*>(ws);
  uint16_t* U = reinterpret_cast<uint16_t*>(base + L.u);
  float* QKV = reinterpret_cast<float*>(base + L.qkv);
  uint16_t* Qr = reinterpret_cast<uint16_t*>(base + L.q);
  uint16_t* Ob = reinterpret_cast<uint16_t*>(base + L.o);
  float* GU = reinterpret_cast<float*>(base + L.gu);
  uint16_t* Mb = reinterpret_cast<uint16_t*>(base + L.m);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int nq = in.n_q_heads, nkv = in.n_kv_heads, F = in.n_cols;
  const int G = D.n_heads / D.n_kv_heads;
  const int64_t fpad = std::max<int64_t>(8, (F + 7) / 8 * 8);
  hipError_t e;
  auto check = [&](const char* what) -> vt_status {
    e = hipGetLastError();
    return e == hipSuccess ? VT_OK : fail(VT_ERR_HIP, "%s launch: %s", what, hipGetErrorString(e));
  };

  if (attn) {
    hipLaunchKernelGGL(pf::rmsnorm_rows_kernel, dim3(n_tok), dim3(pf::RT), 0, s,
                       static_cast<const uint16_t*>(io->x), static_cast<const uint16_t*>(w->g_attn), U,
                       static_cast<int>(H), D.rms_eps);
    if ((st = check("rmsnorm")) != VT_OK) return st;
    {
      // The B operand takes rows from two matrices, so the projection runs
      // as a [Wq; Wk] GEMM and a Wv GEMM into one fp32 buffer.
      pf::GemmArgs a{};
      a.A = U;
      a.lda = H;
      a.K = static_cast<int>(H);
      a.M = n_tok;
      a.B1 = static_cast<const uint16_t*>(w->wq);
      a.ldb1 = w->ld_q;
      a.n1 = nq * static_cast<int>(d);
      a.B2 = static_cast<const uint16_t*>(w->wk);
      a.ldb2 = w->ld_k;
      a.N = (nq + nkv) * static_cast<int>(d);
      if ((st = launch_gemm(a, pf::EpiStoreF32{QKV, (nq + 2 * nkv) * d}, s)) != VT_OK) return st;
      a.B1 = static_cast<const uint16_t*>(w->wv);
      a.ldb1 = w->ld_v;
      a.n1 = nkv * static_cast<int>(d);
      a.B2 = nullptr;
      a.ldb2 = 0;
      a.N = nkv * static_cast<int>(d);
      if ((st = launch_gemm(a, pf::EpiStoreF32{QKV + (nq + nkv) * d, (nq + 2 * nkv) * d}, s)) !=
          VT_OK)
        return st;
      hipLaunchKernelGGL(pf::rope_append_kernel, dim3(n_tok), dim3(pf::RT), 0, s, QKV,
                         static_cast<int>((nq + 2 * nkv) * d), Qr, static_cast<uint16_t*>(kv->k),
                         static_cast<uint16_t*>(kv->v), nq, nkv, static_cast<int>(d), kv->capacity,
                         pos0, D.rope_base);
      if ((st = check("rope_append")) != VT_OK) return st;
      const int blocks = nq * ((n_tok + pf::QB - 1) / pf::QB);
      if (d == 128)
        hipLaunchKernelGGL(pf::attn_prefill_kernel<128>, dim3(blocks), dim3(kWave), 0, s, Qr, Ob,
                           static_cast<const uint16_t*>(kv->k), static_cast<const uint16_t*>(kv->v),
                           n_tok, nq, G, kv->capacity, pos0);
      else
        hipLaunchKernelGGL(pf::attn_prefill_kernel<64>, dim3(blocks), dim3(kWave), 0, s, Qr, Ob,
                           static_cast<const uint16_t*>(kv->k), static_cast<const uint16_t*>(kv->v),
                           n_tok, nq, G, kv->capacity, pos0);
      if ((st = check("attention")) != VT_OK) return st;
    }
    pf::GemmArgs a{};
    a.A = Ob;
    a.lda = std::max<int64_t>(nq * d, 8);
    a.K = nq * static_cast<int>(d);
    a.M = n_tok;
    a.B1 = static_cast<const uint16_t*>(w->wo);
    a.ldb1 = w->ld_o;
    a.n1 = static_cast<int>(H);
    a.N = static_cast<int>(H);
    pf::EpiResidual epi{static_cast<uint16_t*>(io->attn_partial), static_cast<uint16_t*>(io->h),
                        static_cast<const uint16_t*>(io->x),
                        static_cast<const uint16_t*>(io->peer_attn), H};
    if ((st = launch_gemm(a, epi, s)) != VT_OK) return st;
  }
  if (ffn) {
    hipLaunchKernelGGL(pf::rmsnorm_rows_kernel, dim3(n_tok), dim3(pf::RT), 0, s,
                       static_cast<const uint16_t*>(io->h), static_cast<const uint16_t*>(w->g_ffn), U,
                       static_cast<int>(H), D.rms_eps);
    if ((st = check("rmsnorm")) != VT_OK) return st;
    pf::GemmArgs a{};
    a.A = U;
    a.lda = H;
    a.K = static_cast<int>(H);
    a.M = n_tok;
    a.B1 = static_cast<const uint16_t*>(w->wg);
    a.ldb1 = w->ld_g;
    a.n1 = F;
    a.B2 = static_cast<const uint16_t*>(w->wu);
    a.ldb2 = w->ld_u;
    a.N = 2 * F;
    if ((st = launch_gemm(a, pf::EpiStoreF32{GU, 2 * F}, s)) != VT_OK) return st;
    hipLaunchKernelGGL(pf::silu_gate_kernel, dim3(n_tok), dim3(pf::RT), 0, s, GU, 2 * F, Mb, F,
                       static_cast<int>(fpad));
    if ((st = check("silu_gate")) != VT_OK) return st;
    pf::GemmArgs b{};
    b.A = Mb;
    b.lda = fpad;
    b.K = F;
    b.M = n_tok;
    b.B1 = static_cast<const uint16_t*>(w->wd);
    b.ldb1 = w->ld_d;
    b.n1 = static_cast<int>(H);
    b.N = static_cast<int>(H);
    pf::EpiResidual epi{static_cast<uint16_t*>(io->ffn_partial), static_cast<uint16_t*>(io->y),
                        static_cast<const uint16_t*>(io->h),
                        static_cast<const uint16_t*>(io->peer_ffn), H};
    if ((st = launch_gemm(b, epi, s)) != VT_OK) return st;
  }
  if (attn) kv->len = pos0 + n_tok;
  return VT_OK;
}
