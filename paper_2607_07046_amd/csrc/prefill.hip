// Prefill chunk of one device's shard on gfx950 matrix cores.
//
// Paper Sec. 2.1 (LLM Inference): the prompt's tokens are processed in
// parallel and their K and V are accumulated into the KV cache; with the
// tensor-parallel shard of Sec. 3.2.1 each device does its heads and FFN
// columns. For T tokens at positions pos0..pos0+T-1 the projections are
// dense GEMMs (M = T), run here on fp16 MFMA (v_mfma_f32_32x32x16_f16) with
// fp32 accumulation; every elementwise step runs in the epilogue of the
// GEMM that produces its input:
//   rmsnorm_rows   U = fp16(RMSNorm(X) * g_attn), and the rotary angles
//   gemm  QKV      [q | k | v] = U [Wq; Wk; Wv]^T; epilogue: Q = fp16(RoPE(q)
//                  / sqrt(d)), K = fp16(RoPE(k)) and V = fp16(v) into the
//                  cache at positions pos0 + t
//   attn_prefill   O = causal softmax(Q K^T) V, token t sees 0..pos0+t
//   gemm  O        P_attn = O Wo^T; epilogue: H = fp16(X + P_attn + peer),
//                  the FFN input fp16(H * g_ffn) and per-tile sums of H^2
//   gemm  gate/up  G, Up = (H * g_ffn) [Wg | Wu]^T, gate and up rows
//                  interleaved in blocks of 64; epilogue: the RMSNorm's
//                  1 / rms per token from the sums of H^2 scales G and Up,
//                  M = fp16(silu(G) * Up)
//   gemm  down     P_ffn = M Wd^T; epilogue: Y = fp16(H + P_ffn + peer)
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

// Lane-group sums through DPP (no LDS round trip): dpp_xor1 adds lane l ^ 1;
// sum16 leaves every lane of each aligned group of 16 with the group's sum.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float dpp_xor1(float v) { return v + dpp_mov<0xB1>(v); }  // quad_perm [1,0,3,2]
__device__ __forceinline__ float sum16(float v) {
  v = dpp_xor1(v);
  v += dpp_mov<0x4E>(v);   // quad_perm [2,3,0,1]: the quad's sum
  v += dpp_mov<0x141>(v);  // row_half_mirror: the other quad of the 8
  v += dpp_mov<0x140>(v);  // row_mirror: the other 8 of the 16
  return v;
}

// Split sp's share of a tile sum: the own registers for the own split.
__device__ __forceinline__ f32x4 sp_pick(int sp, int split, f32x4 own, f32x4 loaded) {
  return sp == split ? own : loaded;
}

// The 8 halves of w with those at index >= v set to zero.
__device__ __forceinline__ u32x4 zero_past(u32x4 w, int v) {
  w.x = v >= 2 ? w.x : (v >= 1 ? (w.x & 0xFFFFu) : 0u);
  w.y = v >= 4 ? w.y : (v >= 3 ? (w.y & 0xFFFFu) : 0u);
  w.z = v >= 6 ? w.z : (v >= 5 ? (w.z & 0xFFFFu) : 0u);
  w.w = v >= 8 ? w.w : (v >= 7 ? (w.w & 0xFFFFu) : 0u);
  return w;
}

// ---------------------------------------------------------------------------
// Split-K GEMM   C[m][n] = sum over k of A[m][k] * B[n][k]  (fp16 in, fp32
// accumulate), followed by one of four epilogues (EPI_*) that turns the
// 128 x 128 output tile into the layer's next operands. M is the chunk's
// tokens, N the shard's output features, K the input features. A is
// k-step-major (see kmajor) with zeros past K; B is row-major. The weights
// (B) are the large operand and are streamed once; A is small and re-read
// from L2 by every N tile. The K range is cut into ``splits`` slices (the
// count comes from the host's cost model, choose_split) so that short
// chunks still fill the compute units; the slices of a tile meet through a
// counter, and the last to arrive adds them in slice order (a fixed
// summation order) and runs the epilogue.
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
constexpr int TLD = GBN + 4;               // LDS row of the epilogue's fp32 tile
// two B stages in the main loop; the fp32 output tile and a per-token
// factor in the epilogue (two workgroups per compute unit still fit)
constexpr int GEMM_LDS_BYTES = (GBM * TLD + GBM) * 4 > 2 * STAGE * 2 ? (GBM * TLD + GBM) * 4 : 2 * STAGE * 2;
static_assert(2 * GEMM_LDS_BYTES <= 160 * 1024, "two workgroups per compute unit");
constexpr int GEMM_SLOTS = 512;            // two workgroups per compute unit
constexpr int MAX_SPLITS = 4;
constexpr int RASTER_M = 8;                // M tiles per block of an XCD's tile walk
constexpr unsigned kWaitLimit = 1u << 22;  // polls of the split-K wait: far beyond any slice's stores


struct BSrc {
  const uint16_t* p;
  int64_t ld;
  int start, rows;  // virtual rows [start, start + rows); start a multiple of 8
};

// What the last split of an output tile does with the summed tile.
enum { EPI_QKV = 0, EPI_O = 1, EPI_GU = 2, EPI_DOWN = 3 };

struct GemmArgs {
  const uint16_t* A;  // k-step-major, ceil(K / 16) k-steps of M tokens
  BSrc b[3];
  int nb;
  int interleave;     // b[0] and b[1] rows interleaved in blocks of 64 (gate/up)
  float* P;           // split-K partial tiles (fragment order)
  unsigned* cnt;      // per output tile: slices arrived, slices stored (zero at launch)
  unsigned* err;      // the workspace's error word (set if a wait ever times out)
  int M, N, K;
  int m_tiles, n_tiles, splits, kps;  // kps: k-tiles per split
  int epi;
  // epilogue operands (fp16 unless stated; [M][H] row-major)
  int H;
  float eps;
  const uint16_t* base;  // O: x; DOWN: h
  const uint16_t* peer;  // nullable
  uint16_t* partial;     // O: attention partial; DOWN: FFN partial
  uint16_t* out;         // O: h; DOWN: y (nullable)
  const uint16_t* gain;  // O: g_ffn when the FFN follows (else NULL)
  uint16_t* U;           // O: FFN input fp16(h * g_ffn), k-step-major
  float* rowsq;          // O: [M][n_tiles] sums of h^2 over each tile's columns; GU: read (NULL: 1 / rms = 1)
  int rowsq_tiles;       // GU: column tiles of the O GEMM
  uint16_t *Q, *kc, *vc; // QKV outputs: Q [M][nq][d], the KV cache [n_kv][cap][d]
  const float* rope;     // [M][d / 2][2] cos, sin of each rotary angle
  int nq, nkv, d, cap, pos0;
  uint16_t* Mo;          // GU: fp16(silu(G) * Up), k-step-major, kpad columns
  int F, kpad;
};

__global__ void __launch_bounds__(GT, 2) gemm_kernel(GemmArgs g) {
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
  // Workgroups with equal index mod 8 run on one XCD. An XCD takes every
  // eighth (N tile, split) unit and walks its tiles in blocks of up to
  // RASTER_M M tiles x all its units, M tile fastest: the M tiles of one
  // unit run together (its B slice comes into that XCD's L2 once), and with
  // many M tiles the workgroups resident at once still share each
  // activation k-slab across all the XCD's units instead of re-reading the
  // whole of A for every few units (4096-token chunk: 1.31 -> 1.21 ms).
  const int id = blockIdx.x;
  const int groups = (g.n_tiles * g.splits + 7) / 8;  // units per XCD (at most)
  const int j = id / 8;
  const int bm = min(g.m_tiles, RASTER_M);
  const int blk = j / (bm * groups);
  const int rows = min(bm, g.m_tiles - blk * bm);  // M tiles in this block
  const int r = j - blk * bm * groups;
  const int unit = (r / rows) * 8 + id % 8;
  const int m_tile = blk * bm + r % rows;
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
    const int n = n0 + (t + u * GT) / 8;
    int j = 2, r;
    if (g.interleave) {  // blocks of 64 rows alternate between b[0] and b[1]
      j = (r0 / 64) % 2;
      r = (n / 128) * 64 + n % 64;
    } else {
      if (r0 < g.b[1].start || g.nb < 2) j = 0;
      else if (r0 < g.b[2].start || g.nb < 3) j = 1;
      r = n - (j == 0 ? g.b[0].start : (j == 1 ? g.b[1].start : g.b[2].start));
    }
    const BSrc src = j == 0 ? g.b[0] : (j == 1 ? g.b[1] : g.b[2]);
    rsel[u] = j == 0 ? rs[0] : (j == 1 ? rs[1] : rs[2]);
    boff[u] = (n < g.N && r >= 0 && r < src.rows) ? static_cast<uint32_t>(r * src.ld * 2) : kOOB;
  }
  auto load_b = [&](int kt, u32x4 (&vb)[B_CH]) {  // k-tile kt (absolute)
    const int k = kt * GBK + ccol;
    const uint32_t out = (kt < kt_end && k < g.K) ? 0u : kOOB;
#pragma unroll
    for (int u = 0; u < B_CH; ++u)
      vb[u] = buf_load16(rsel[u], (boff[u] + static_cast<uint32_t>(k) * 2u) | out | (boff[u] & kOOB));
  };
  // k-tile kt into LDS; a chunk that straddles K keeps only its columns
  // below K (the row padding past K may hold anything)
  auto store_b = [&](uint16_t* st, u32x4 (&vb)[B_CH], int kt) {
    if (g.K & 7) {
      const int v = g.K - (kt * GBK + ccol);
#pragma unroll
      for (int u = 0; u < B_CH; ++u) vb[u] = zero_past(vb[u], v);
    }
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
  // The next k-tile's B chunks go to the other LDS stage in the middle of
  // the k-tile (after the second k-step's MFMAs are issued), so the LDS
  // writes overlap the matrix cores instead of following them.
  auto compute = [&](const uint16_t* st, int ks_base, int s0, uint16_t* st_next, u32x4 (&vb)[B_CH], int kt_next) {
    u32x4 bf[2][4];
    read_b(st, 0, bf[0]);
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      if (ks + 1 < KSTEPS) read_b(st, ks + 1, bf[(ks + 1) & 1]);
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[b] = mfma32(ar[s0 + ks], bf[ks & 1][b], acc[b]);
      load_a(ks_base + ks + RING, ar[s0 + ks]);
      if (ks == 1) store_b(st_next, vb, kt_next);
    }
  };

  uint16_t* L0 = lds;
  uint16_t* L1 = lds + STAGE;
  u32x4 rb0[B_CH], rb1[B_CH];
#pragma unroll
  for (int s = 0; s < RING; ++s) load_a(s, ar[s]);
  load_b(kt0, rb0);
  load_b(kt0 + 1, rb1);
  store_b(L0, rb0, kt0);
  __syncthreads();
  // two k-tiles per trip; an odd count runs one all-zero tile at the end
  // (the scheduling barriers keep the B prefetch ahead of the MFMAs)
  for (int i = 0; i < nkt; i += 2) {
    load_b(kt0 + i + 2, rb0);
    __builtin_amdgcn_sched_barrier(0);
    compute(L0, i * KSTEPS, 0, L1, rb1, kt0 + i + 1);
    __syncthreads();
    load_b(kt0 + i + 3, rb1);
    __builtin_amdgcn_sched_barrier(0);
    compute(L1, (i + 1) * KSTEPS, KSTEPS, L0, rb0, kt0 + i + 2);
    __syncthreads();
  }

  // Split-K: the slices of a tile take arrival tickets when their k range
  // is done. All but the last to arrive park their sums in their slot of
  // the partial buffer (fragment order: each lane's 64 values as 16
  // contiguous 16-byte chunks, chunk-major over the workgroup, so each
  // store and load instruction moves 4 KiB contiguously) and count
  // themselves stored; the last waits for those stores, which are already
  // under way (every slice it waits for has arrived, so is running), adds
  // the slices in slice order (its own from registers: the order, and so
  // the result, does not depend on which slice arrives last) and runs the
  // epilogue. Tiles cross XCDs through the agent-scope coherent path.
  // The epilogue's global inputs (rotary table rows; residual base and
  // peer rows and the FFN gain; the tokens' partial sums of squares) are
  // loaded ahead of the split-K wait and reduction, so their round trip
  // overlaps those. Thread t takes features f..f+7 (f = 8 (t%16)) of tokens
  // t / 16 + 16 j of the tile; for the gate/up epilogue, the first RQ
  // partial sums of half t % 2 of token t / 2.
  constexpr int RJ = GBM / 16;
  const int ef = 8 * (t % 16), en = n0 + ef;
  const int qd = g.nq * g.d, kd = g.nkv * g.d;
  constexpr int RQ = 16;
  const int nt = g.rowsq_tiles, half = t % 2;
  const int q0 = half * ((nt + 1) / 2), q1 = half ? nt : (nt + 1) / 2;
  u32x4 pre[2 * RJ], pre_g;
  auto prefetch = [&]() {
    if (g.epi == EPI_QKV) {
      if (en < g.N && en < qd + kd) {
        const int c = (en < qd ? en : en - qd) % g.d;
#pragma unroll
        for (int j = 0; j < RJ; ++j) {
          const int m = m0 + t / 16 + 16 * j;
          if (m < g.M) {
            const float* cs = g.rope + (static_cast<int64_t>(m) * (g.d / 2) + c / 2) * 2;
            pre[2 * j] = *reinterpret_cast<const u32x4*>(cs);
            pre[2 * j + 1] = *reinterpret_cast<const u32x4*>(cs + 4);
          }
        }
      }
    } else if (g.epi == EPI_O || g.epi == EPI_DOWN) {
      if (en < g.N) {
#pragma unroll
        for (int j = 0; j < RJ; ++j) {
          const int m = m0 + t / 16 + 16 * j;
          const int64_t e = static_cast<int64_t>(m) * g.H + en;
          if (m < g.M) {
            pre[j] = load16(g.base + e);
            if (g.peer) pre[RJ + j] = load16(g.peer + e);
          }
        }
        if (g.epi == EPI_O && g.gain) pre_g = load16(g.gain + en);
      }
    } else if (g.rowsq) {  // EPI_GU
      const int m = m0 + t / 2;
      if (m < g.M) {
        float* rq = reinterpret_cast<float*>(pre);
#pragma unroll
        for (int k = 0; k < RQ; ++k)
          if (q0 + k < q1) rq[k] = g.rowsq[static_cast<int64_t>(m) * nt + q0 + k];
      }
    }
  };

  if (g.splits > 1) {
    __shared__ unsigned ticket;
    const int tile = m_tile * g.n_tiles + n_tile;
    unsigned* arrived = g.cnt + 2 * tile;
    unsigned* stored = arrived + 1;
    const int64_t tile_floats = static_cast<int64_t>(GBM) * GBN;
    const uint32_t tile_bytes = static_cast<uint32_t>(tile_floats * 4);
    auto slot = [&](int sp) {
      return make_rsrc(g.P + (static_cast<int64_t>(sp) * g.m_tiles * g.n_tiles + tile) * tile_floats,
                       sp < g.splits ? tile_bytes : 0u);
    };
    auto chunk_off = [&](int c) { return static_cast<uint32_t>(((c * GT) + t) * 16); };
    if (t == 0) ticket = __hip_atomic_fetch_add(arrived, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    if (ticket != static_cast<unsigned>(g.splits - 1)) {
      const rsrc_t mine = slot(split);
#pragma unroll
      for (int c = 0; c < 16; ++c) {
        const f32x4 v = f32x4{acc[c / 4][4 * (c % 4)], acc[c / 4][4 * (c % 4) + 1], acc[c / 4][4 * (c % 4) + 2],
                              acc[c / 4][4 * (c % 4) + 3]};
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), mine, chunk_off(c), 0, kCoherent);
      }
      mem_done();
      __syncthreads();
      if (t == 0) __hip_atomic_fetch_add(stored, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return;
    }
    prefetch();
    if (t == 0) {
      unsigned n = 0;
      while (__hip_atomic_load(stored, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) <
             static_cast<unsigned>(g.splits - 1)) {
        __builtin_amdgcn_s_sleep(1);
        if (++n > kWaitLimit) {  // never expected: report instead of hanging
          __hip_atomic_fetch_or(g.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          break;
        }
      }
    }
    __syncthreads();
    // At most MAX_SPLITS slices; those past g.splits read zero (an empty
    // range) and are added last, which leaves the sum unchanged. A quarter
    // of the tile at a time, every load is issued before the first add, so
    // the slices' data arrive in one memory round trip per quarter.
    rsrc_t sr[MAX_SPLITS];
#pragma unroll
    for (int sp = 0; sp < MAX_SPLITS; ++sp) sr[sp] = slot(sp);
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      f32x4 v[4][MAX_SPLITS];
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int sp = 0; sp < MAX_SPLITS; ++sp)
          v[c][sp] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                   sr[sp], sp == split ? kOOB : chunk_off(4 * h + c), 0, kCoherent));
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int cc = 4 * h + c;
        const f32x4 own = f32x4{acc[cc / 4][4 * (cc % 4)], acc[cc / 4][4 * (cc % 4) + 1],
                                acc[cc / 4][4 * (cc % 4) + 2], acc[cc / 4][4 * (cc % 4) + 3]};
        f32x4 sum = sp_pick(0, split, own, v[c][0]);
#pragma unroll
        for (int sp = 1; sp < MAX_SPLITS; ++sp) sum += sp_pick(sp, split, own, v[c][sp]);
        acc[cc / 4][4 * (cc % 4)] = sum.x;
        acc[cc / 4][4 * (cc % 4) + 1] = sum.y;
        acc[cc / 4][4 * (cc % 4) + 2] = sum.z;
        acc[cc / 4][4 * (cc % 4) + 3] = sum.w;
      }
    }
  } else {
    prefetch();
  }

  // The summed tile goes through LDS (fp32, rows of TLD floats) so that the
  // epilogue reads rows of 8 consecutive features per thread: every global
  // access below is one 16-byte load or store, and 16 consecutive threads
  // cover one token's 128 features.
  // Accumulator i of tile b: token 8(i/4) + 4(l/32) + i%4 of the wave's 32,
  // feature b * 32 + l%32.
  float* tl = reinterpret_cast<float*>(lds);
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int i = 0; i < 16; ++i)
      tl[(wave * 32 + 8 * (i / 4) + 4 * (lane / 32) + i % 4) * TLD + b * 32 + lane % 32] = acc[b][i];
  __syncthreads();
  // k-step-major outputs (the next GEMM's activation operand) are staged as
  // fp16 in the first half of each token's LDS row and then copied out with
  // consecutive threads on consecutive tokens, so each k-step's 16 features
  // of the tile's tokens leave as one contiguous run. A thread's staging
  // store lands on floats that lanes of its own wave read in the same
  // straight-line code just before, so only threads that have read their
  // row may stage into it: the zero padding past the last valid feature
  // (valid is a multiple of 8) is written at copy time, not staged.
  auto stage8 = [&](int mm, int f, u32x4 v) {
    *reinterpret_cast<u32x4*>(reinterpret_cast<uint16_t*>(tl + mm * TLD) + f) = v;
  };
  auto copy_kmajor = [&](uint16_t* dst, int groups, int col0, int limit, int valid) {
    __syncthreads();
    for (int q = t / GBM; q < groups; q += GT / GBM) {
      const int mm = t % GBM, m = m0 + mm, col = col0 + 16 * q;
      if (m < g.M && col < limit) {
        const uint16_t* src = reinterpret_cast<const uint16_t*>(tl + mm * TLD) + 16 * q;
        uint16_t* o = dst + kmajor(col, m, g.M);
        *reinterpret_cast<u32x4*>(o) = *reinterpret_cast<const u32x4*>(src);
        *reinterpret_cast<u32x4*>(o + 8) =
            col + 8 < valid ? *reinterpret_cast<const u32x4*>(src + 8) : u32x4{0u, 0u, 0u, 0u};
      }
    }
  };
  auto row8 = [&](int mm, int f, float (&v)[8]) {
    const f32x4 lo = *reinterpret_cast<const f32x4*>(tl + mm * TLD + f);
    const f32x4 hi = *reinterpret_cast<const f32x4*>(tl + mm * TLD + f + 4);
    v[0] = lo.x; v[1] = lo.y; v[2] = lo.z; v[3] = lo.w;
    v[4] = hi.x; v[5] = hi.y; v[6] = hi.z; v[7] = hi.w;
  };

  if (g.epi == EPI_QKV) {
    // features f..f+7 of one head; rotary pairs (2c, 2c+1) are adjacent
    const int f = ef, n = en;
    if (n < g.N) {
      const bool rot = n < qd + kd;
      const int c = (n < qd ? n : n - qd) % g.d;
      const float sc = n < qd ? 1.0f / sqrtf(static_cast<float>(g.d)) : 1.f;
#pragma unroll
      for (int j = 0; j < RJ; ++j) {
        const int mm = t / 16 + 16 * j, m = m0 + mm;
        if (m >= g.M) break;
        float v[8];
        row8(mm, f, v);
        uint16_t h[8];
        if (rot) {
          const f32x4 r0 = __builtin_bit_cast(f32x4, pre[2 * j]), r1 = __builtin_bit_cast(f32x4, pre[2 * j + 1]);
          const float co[4] = {r0.x, r0.z, r1.x, r1.z}, si[4] = {r0.y, r0.w, r1.y, r1.w};
#pragma unroll
          for (int p = 0; p < 4; ++p) {
            h[2 * p] = f2h((v[2 * p] * co[p] - v[2 * p + 1] * si[p]) * sc);
            h[2 * p + 1] = f2h((v[2 * p] * si[p] + v[2 * p + 1] * co[p]) * sc);
          }
          uint16_t* dst = n < qd ? g.Q + (static_cast<int64_t>(m) * g.nq + n / g.d) * g.d + c
                                 : g.kc + (static_cast<int64_t>((n - qd) / g.d) * g.cap + g.pos0 + m) * g.d + c;
          *reinterpret_cast<u32x4*>(dst) = pack8(h);
        } else {
          const int nv = n - qd - kd;
#pragma unroll
          for (int e = 0; e < 8; ++e) h[e] = f2h(v[e]);
          *reinterpret_cast<u32x4*>(g.vc + (static_cast<int64_t>(nv / g.d) * g.cap + g.pos0 + m) * g.d + nv % g.d) =
              pack8(h);
        }
      }
    }
  } else if (g.epi == EPI_O || g.epi == EPI_DOWN) {
    // partial = fp16(p); out = fp16(base + p + peer); for O with the FFN to
    // follow also the FFN input fp16(out * g_ffn) and each token's sum of
    // out^2 over this tile's 128 columns (the RMSNorm is finished by the
    // gate/up epilogue)
    const bool norm = g.epi == EPI_O && g.gain;
    const int f = ef, n = en;
    const int hpad = (g.H + 15) / 16 * 16;
    const bool in = n < g.N;
    float gg[8];
    if (norm && in) unpack8(pre_g, gg);
#pragma unroll
    for (int j = 0; j < RJ; ++j) {
      const int mm = t / 16 + 16 * j, m = m0 + mm;
      if (m >= g.M) break;  // uniform over each group of 16 threads
      float sq = 0.f;
      if (in) {
        float v[8], b[8], pe[8];
        row8(mm, f, v);
        const int64_t e = static_cast<int64_t>(m) * g.H + n;
        unpack8(pre[j], b);
        if (g.peer) unpack8(pre[RJ + j], pe);
        uint16_t ph[8], oh[8], uh[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          ph[k] = f2h(v[k]);
          oh[k] = f2h(b[k] + v[k] + (g.peer ? pe[k] : 0.f));
          if (norm) {
            const float o = h2f(oh[k]);
            sq = fmaf(o, o, sq);
            uh[k] = f2h(o * gg[k]);
          }
        }
        *reinterpret_cast<u32x4*>(g.partial + e) = pack8(ph);
        if (g.out) *reinterpret_cast<u32x4*>(g.out + e) = pack8(oh);
        if (norm) stage8(mm, f, pack8(uh));
      }
      if (norm) {
        sq = sum16(sq);
        if (t % 16 == 0) g.rowsq[static_cast<int64_t>(m) * g.n_tiles + n_tile] = sq;
      }
    }
    if (norm) copy_kmajor(g.U, GBN / 16, n0, hpad, g.H);
  } else {  // EPI_GU: tile features 0..63 gate and 64..127 up of the same 64 columns
    float* rinv = tl + GBM * TLD;  // 1 / rms of the tile's tokens
    if (g.rowsq) {
      // thread t: token t / 2 of the tile, column tiles q0..q1-1 (half t % 2)
      const int mm = t / 2, m = m0 + mm;
      float ss = 0.f;
      if (m < g.M) {
        const float* rq = reinterpret_cast<const float*>(pre);
#pragma unroll
        for (int k = 0; k < RQ; ++k)
          if (q0 + k < q1) ss += rq[k];
        for (int k = q0 + RQ; k < q1; ++k) ss += g.rowsq[static_cast<int64_t>(m) * nt + k];
      }
      ss = dpp_xor1(ss);
      if (half == 0) rinv[mm] = 1.0f / sqrtf(ss / static_cast<float>(g.H) + g.eps);
    } else if (t < GBM) {
      rinv[t] = 1.f;
    }
    __syncthreads();
    const int f = 8 * (t % 8), col0 = (n0 / 128) * 64, col = col0 + f;
    if (col < g.kpad) {
#pragma unroll 2
      for (int j = 0; j < GBM / 32; ++j) {
        const int mm = t / 8 + 32 * j, m = m0 + mm;
        if (m >= g.M) break;
        float gt[8], up[8];
        row8(mm, f, gt);
        row8(mm, 64 + f, up);
        const float r = rinv[mm];
        uint16_t h[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const float a = gt[k] * r;
          h[k] = f2h(a / (1.0f + __expf(-a)) * (up[k] * r));
        }
        stage8(mm, f, pack8(h));
      }
    }
    copy_kmajor(g.Mo, 4, col0, g.kpad, g.kpad);
  }
}

// ---------------------------------------------------------------------------
// row-wise helpers
// ---------------------------------------------------------------------------
constexpr int RT = 256;

// U[t] = fp16(X[t] / sqrt(mean(X[t]^2) + eps) * g), one workgroup per row
// (grid = the chunk's tokens); U is k-step-major. The chunk's first kernel:
// it also zeroes the GEMMs' ncnt split-K counters and, when rope is not
// NULL, writes the rotary (cos, sin) of pair i at position pos0 + t to
// rope[t][i] (the QKV epilogue reads them).
__global__ void __launch_bounds__(RT) rmsnorm_rows_kernel(const uint16_t* X, const uint16_t* g,
                                                          uint16_t* U, int H, float eps, unsigned* cnt,
                                                          int ncnt, float* rope, int d, int pos0,
                                                          float base) {
  __shared__ float red[RT / kWave];
  const int t = blockIdx.x, M = gridDim.x;
  for (int i = t * RT + threadIdx.x; i < ncnt; i += M * RT) cnt[i] = 0u;
  if (rope && static_cast<int>(threadIdx.x) < d / 2) {
    float c, s;
    rope_angle(pos0 + t, threadIdx.x, d, base, c, s);
    *reinterpret_cast<float2*>(rope + (static_cast<int64_t>(t) * (d / 2) + threadIdx.x) * 2) = make_float2(c, s);
  }
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
// lane) is gathered with two transposing 8-byte LDS reads. The 32 queries are staged
// in LDS once per workgroup (every wave multiplies the same Q block), which
// keeps the loop's registers within two waves per SIMD. Apart from reading
// Q, a wave only touches its own LDS region inside the loop, so the loop
// needs no workgroup barrier.
// The output O (the O projection's input) is written k-step-major.
// ---------------------------------------------------------------------------
constexpr int QB = 32, KB = 32, AW = 8;

typedef short v4h16 __attribute__((ext_vector_type(4)));

// 4 fp16 values per lane from LDS, transposed within each group of 16 lanes
// (ds_read_b64_tr_b16: lane j supplies the 8-byte address of its 4 values;
// lane i receives value i % 4 of lanes i / 4, 4 + i / 4, 8 + i / 4 and
// 12 + i / 4 of its group).
__device__ __forceinline__ v4h16 lds_read_tr16(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4h16*)(p));
}

__device__ __forceinline__ u32x4 pack_v4(v4h16 a, v4h16 b) {
  auto w = [](short x, short y) {
    return static_cast<unsigned>(static_cast<uint16_t>(x)) | (static_cast<unsigned>(static_cast<uint16_t>(y)) << 16);
  };
  return u32x4{w(a.x, a.y), w(a.z, a.w), w(b.x, b.y), w(b.z, b.w)};
}

__device__ __forceinline__ int swap_bits23(int r) {
  return (r & ~0xC) | ((r & 4) << 1) | ((r & 8) >> 1);
}

template <int D>
struct AttnLds {
  static constexpr int KLD = D + 8;   // row stride of the K and V tiles (halves)
  static constexpr int OLD = D + 4;   // row stride of a wave's fp32 output in the merge
  static constexpr int WAVE_HALVES = 2 * KB * KLD;
  static constexpr int Q_HALVES = QB * KLD;  // the workgroup's Q block (rows of KLD)
  static_assert(WAVE_HALVES * 2 >= (QB * OLD + 2 * QB) * 4, "merge buffer must fit a wave's region");
};

template <int D>
__global__ void __launch_bounds__(AW * kWave) attn_prefill_kernel(const uint16_t* Q, uint16_t* O,
                                                                  const uint16_t* kc, const uint16_t* vc,
                                                                  int T, int nq, int G, int cap, int pos0,
                                                                  int window) {
  using LY = AttnLds<D>;
  constexpr int KLD = LY::KLD, OLD = LY::OLD;
  __shared__ __attribute__((aligned(16))) uint16_t smem[AW * LY::WAVE_HALVES + LY::Q_HALVES];
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

  // the Q block into LDS (queries past T repeat the last one); the Q^T
  // operand of k-step ks: lane supplies Q[tq][16 ks + 8 (l/32) + e]
  uint16_t* Qs = smem + AW * LY::WAVE_HALVES;
  for (int c = threadIdx.x; c < QB * D / 8; c += AW * kWave) {
    const int q = c / (D / 8), col = (c % (D / 8)) * 8;
    const int tqc = min(t0 + q, T - 1);
    *reinterpret_cast<u32x4*>(Qs + q * KLD + col) = load16(Q + (static_cast<int64_t>(tqc) * nq + j) * D + col);
  }
  __syncthreads();
  auto qfrag = [&](int ks) {
    return *reinterpret_cast<const u32x4*>(Qs + (lane % 32) * KLD + ks * 16 + 8 * (lane / 32));
  };
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
  // Key block kb's chunks into registers through buffer ranges that end
  // after last_key: positions past it (never attended) read as zero, and
  // the block is fetched in one round trip. Chunk u of this lane: key
  // (lane + 64 u) / (D/8) of the block, 8 dimensions from col; its byte
  // offset within the block and its LDS offsets do not depend on the block.
  const uint32_t range = static_cast<uint32_t>(last_key + 1) * D * 2u;
  const rsrc_t rk = make_rsrc(kbase, range), rv = make_rsrc(vbase, range);
  uint32_t goff[CPL];
  int kst[CPL], vst[CPL];
#pragma unroll
  for (int u = 0; u < CPL; ++u) {
    const int c = lane + u * kWave;
    const int key = c / (D / 8), col = (c % (D / 8)) * 8;
    goff[u] = static_cast<uint32_t>(key * D + col) * 2u;
    kst[u] = swap_bits23(key) * KLD + col;
    vst[u] = key * KLD + col;
  }
  u32x4 kreg[CPL], vreg[CPL];
  auto fetch = [&](int kb) {
    const uint32_t base = static_cast<uint32_t>(kb * KB) * D * 2u;
#pragma unroll
    for (int u = 0; u < CPL; ++u) {
      kreg[u] = buf_load16(rk, base + goff[u]);
      vreg[u] = buf_load16(rv, base + goff[u]);
    }
  };
  fetch(min(kb0 + wave, nkb - 1));
  for (int kb = kb0 + wave; kb < nkb; kb += AW) {
    const int p0 = kb * KB;
    // stage K (rows permuted) and V (row-major), then start the next block
#pragma unroll
    for (int u = 0; u < CPL; ++u) {
      *reinterpret_cast<u32x4*>(Ks + kst[u]) = kreg[u];
      *reinterpret_cast<u32x4*>(Vs + vst[u]) = vreg[u];
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
      s = mfma32(kf, qfrag(ks), s);
    }
    // accumulator i: LDS row 8(i/4) + 4(l/32) + i%4 holds key p0 + swap_bits23(row).
    // Only a block that reaches past the block's first query, lies partly
    // outside a sliding window, or serves queries past T masks anything;
    // every other block skips the per-element tests (same values).
    const bool masked = p0 + KB - 1 > pos0 + t0 || t0 + QB > T ||
                        (window > 0 && p0 <= pos0 + t0 + QB - 1 - window);
    float bm = -INFINITY;
    if (masked) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int key = swap_bits23(8 * (i / 4) + 4 * (lane / 32) + i % 4);
        if (p0 + key > qpos || tq >= T || (window > 0 && p0 + key <= qpos - window)) s[i] = -INFINITY;
        bm = fmaxf(bm, s[i]);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i) bm = fmaxf(bm, s[i]);
    }
    bm = fmaxf(bm, __shfl_xor(bm, 32, kWave));
    const float mnew = fmaxf(mrun, bm);
    const float alpha = mrun == -INFINITY ? 0.f : __expf(mrun - mnew);
    float ps = 0.f;
    uint16_t ph[16];
    if (masked) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float e = s[i] == -INFINITY ? 0.f : __expf(s[i] - mnew);
        ps += e;
        ph[i] = f2h(e);
      }
    } else {  // no score is -inf here, and mnew is finite
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float e = __expf(s[i] - mnew);
        ps += e;
        ph[i] = f2h(e);
      }
    }
    ps += __shfl_xor(ps, 32, kWave);
    lrun = lrun * alpha + ps;
    mrun = mnew;
    // o is rescaled only if some query's running maximum moved (an alpha of
    // exactly 1 changes nothing), and not on the wave's first block (o is
    // still zero)
    if (kb != kb0 + wave && __builtin_amdgcn_ballot_w64(alpha != 1.f) != 0) {
#pragma unroll
      for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[mt][i] *= alpha;
    }
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
    // 32 mt + l%32 of keys 16 s2 + 8 (l/32) .. +7, gathered from the
    // row-major V tile by two transposing LDS reads: in each group of 16
    // lanes, lane j reads the 4 dimensions 4 (j%4) .. of key j / 4 and lane
    // i receives dimension i of the 4 keys
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        const int grp = lane / 16, j = lane % 16;
        const uint16_t* vp = Vs + (s2 * 16 + 8 * (grp / 2) + j / 4) * KLD + mt * 32 + 16 * (grp % 2) + 4 * (j % 4);
        const v4h16 lo = lds_read_tr16(vp), hi = lds_read_tr16(vp + 4 * KLD);
        o[mt] = mfma32(pack_v4(lo, hi), pf[s2], o[mt]);
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

// Split-K choice of a GEMM: the slice count S (whole k-tiles each, at most
// MAX_SPLITS, the in-kernel reduction's width) with the smallest modelled
// time. The tiles x S workgroups run in rounds of GEMM_SLOTS (two per compute
// unit); a round in which compute units hold two workgroups advances each by
// one k-tile per kTwoPerCu microseconds, a last round of at most one per
// compute unit per kOnePerCu; each of the (S - 1) x tiles fp32 partial tiles
// costs kPartial (64 KiB stored and read back at about 7 TB/s). The
// constants are MI355X measurements of this kernel on the 7B shapes (the
// per-k-tile rates from the 4096-token chunk's GEMMs, which the model then
// reproduced within 5%, the partial-tile cost from the chip's copy rate). It
// takes fewer slices than a rule of about two rounds of workgroups: at 256
// tokens 2 instead of 4 for QKV (the same time, 2.5 times less partial-tile
// traffic), and at 512 / 1024 / 2048 tokens per chunk 0.222 / 0.340 /
// 0.609 ms against 0.248 / 0.388 / 0.691 for that rule.
struct Split {
  int m_tiles, n_tiles, splits, kps;
};

constexpr double kTwoPerCu = 1.33, kOnePerCu = 0.75, kPartial = 0.0187;

Split choose_split(int M, int N, int K) {
  Split s{};
  s.m_tiles = (M + pf::GBM - 1) / pf::GBM;
  s.n_tiles = (N + pf::GBN - 1) / pf::GBN;
  const int KT = std::max(1, (K + pf::GBK - 1) / pf::GBK);
  const int64_t tiles = std::max(1, s.m_tiles * s.n_tiles);
  double best = 0.0;
  for (int want = 1; want <= std::min(KT, pf::MAX_SPLITS); ++want) {
    const int kps = (KT + want - 1) / want;
    const int splits = (KT + kps - 1) / kps;
    const int64_t groups = tiles * splits;
    const int64_t full = groups / pf::GEMM_SLOTS, rest = groups % pf::GEMM_SLOTS;
    double t = static_cast<double>(full) * kps * kTwoPerCu;
    if (rest > pf::GEMM_SLOTS / 2) t += kps * kTwoPerCu;
    else if (rest > 0) t += kps * kOnePerCu;
    t += static_cast<double>(splits - 1) * static_cast<double>(tiles) * kPartial;
    if (want == 1 || t < best) {
      best = t;
      s.kps = kps;
      s.splits = splits;
    }
  }
  return s;
}

// The shard's prefill GEMMs for T tokens: QKV, O, gate/up, down. N counts
// virtual rows of B: the QKV GEMM's k rows start at the 8-aligned row after
// the q rows (likewise v), and the gate/up GEMM interleaves gate and up rows
// in blocks of 64 (so one output tile holds the gate and up values of the
// same 64 columns).
struct PrefillGemms {
  int M, N[4], K[4];
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
  g.N[2] = (in.n_cols + 63) / 64 * 128;
  g.K[2] = H;
  g.N[3] = H;
  g.K[3] = in.n_cols;
  return g;
}

struct PrefillWs {
  size_t u, q, o, m, part, cnt, rowsq, rope, total;
  int cnt_off[4], ncnt;
};

inline int64_t rup(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

PrefillWs prefill_layout(const vt_shard_spec& s, int32_t T) {
  const vt_shard_info& in = s.info;
  const int64_t H = s.dims.hidden, d = s.dims.head_dim;
  const PrefillGemms gm = prefill_gemms(s, T);
  PrefillWs w{};
  int64_t part = 0;  // one region serves the four GEMMs' split-K tiles in turn
  w.ncnt = 0;
  for (int i = 0; i < 4; ++i) {
    const Split sp = choose_split(gm.M, gm.N[i], gm.K[i]);
    const int64_t tiles = static_cast<int64_t>(sp.m_tiles) * sp.n_tiles;
    if (sp.splits > 1) part = std::max<int64_t>(part, sp.splits * tiles * pf::GBM * pf::GBN * 4);
    w.cnt_off[i] = w.ncnt;
    w.ncnt += 2 * static_cast<int>(tiles);  // arrived, stored
  }
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
  w.cnt = take(4 * static_cast<int64_t>(w.ncnt));
  w.rowsq = take(4 * T * ((H + pf::GBN - 1) / pf::GBN));
  w.rope = take(4 * T * d);
  w.total = off;
  return w;
}

// Launches the split-K GEMM with its epilogue; P holds the split-K tiles and
// cnt the per-tile arrival counters (zero at launch).
vt_status launch_gemm(pf::GemmArgs a, float* P, unsigned* cnt, unsigned* err, hipStream_t s) {
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
  a.cnt = cnt;
  a.err = err;
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

}  // namespace

// Enough for every chunk of 1..max_tokens tokens: the split-K region depends
// on the chunk only through its number of 128-row tiles and may shrink as
// chunks grow (fewer slices), so the layout is taken at the longest chunk of
// each tile count and the largest total kept.
size_t prefill_workspace_bytes(const vt_shard_spec& s, int32_t max_tokens, int32_t) {
  size_t most = 0;
  for (int64_t hi = pf::GBM;; hi += pf::GBM) {
    const int32_t T = static_cast<int32_t>(std::min<int64_t>(hi, max_tokens));
    most = std::max(most, prefill_layout(s, T).total);
    if (T == max_tokens) break;
  }
  return most;
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
  unsigned* cnt = reinterpret_cast<unsigned*>(base + L.cnt);
  float* rowsq = reinterpret_cast<float*>(base + L.rowsq);
  float* rope = reinterpret_cast<float*>(base + L.rope);
  unsigned* err = reinterpret_cast<unsigned*>(base + VT_WS_ERROR_WORD);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int nq = in.n_q_heads, nkv = in.n_kv_heads, F = in.n_cols;
  const int G = D.n_heads / D.n_kv_heads;
  const PrefillGemms gm = prefill_gemms(*spec, n_tok);
  auto check = [&](const char* what) -> vt_status {
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? VT_OK : fail(VT_ERR_HIP, "%s launch: %s", what, hipGetErrorString(e));
  };
  auto gemm = [&](int i, const uint16_t* A, int epi) {
    pf::GemmArgs a{};
    a.A = A;
    a.M = n_tok;
    a.N = gm.N[i];
    a.K = gm.K[i];
    a.epi = epi;
    a.H = static_cast<int>(H);
    a.eps = D.rms_eps;
    return a;
  };

  if (attn) {
    // RMSNorm of x, the rotary table, zeroed split-K counters
    hipLaunchKernelGGL(pf::rmsnorm_rows_kernel, dim3(n_tok), dim3(pf::RT), 0, s,
                       static_cast<const uint16_t*>(io->x), static_cast<const uint16_t*>(w->g_attn), U,
                       static_cast<int>(H), D.rms_eps, cnt, L.ncnt, rope, static_cast<int>(d), pos0,
                       D.rope_base);
    if ((st = check("rmsnorm")) != VT_OK) return st;
    // QKV; epilogue: RoPE, Q, and the append of K and V at pos0..
    pf::GemmArgs a = gemm(0, U, pf::EPI_QKV);
    const int qd = nq * static_cast<int>(d), kd = nkv * static_cast<int>(d);
    a.b[0] = bsrc(w->wq, w->ld_q, 0, qd);
    a.b[1] = bsrc(w->wk, w->ld_k, qd, kd);
    a.b[2] = bsrc(w->wv, w->ld_v, qd + kd, kd);
    a.nb = 3;
    a.Q = Qr;
    a.kc = static_cast<uint16_t*>(kv->k);
    a.vc = static_cast<uint16_t*>(kv->v);
    a.rope = rope;
    a.nq = nq;
    a.nkv = nkv;
    a.d = static_cast<int>(d);
    a.cap = kv->capacity;
    a.pos0 = pos0;
    if ((st = launch_gemm(a, P, cnt + L.cnt_off[0], err, s)) != VT_OK) return st;
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
    // O; epilogue: h = x + p_attn + peer, and with the FFN to follow its
    // input h * g_ffn and the sums of h^2 its RMSNorm needs
    pf::GemmArgs o = gemm(1, Ob, pf::EPI_O);
    o.b[0] = bsrc(w->wo, w->ld_o, 0, gm.N[1]);
    o.nb = 1;
    o.base = static_cast<const uint16_t*>(io->x);
    o.peer = static_cast<const uint16_t*>(io->peer_attn);
    o.partial = static_cast<uint16_t*>(io->attn_partial);
    o.out = static_cast<uint16_t*>(io->h);
    if (ffn) {
      o.gain = static_cast<const uint16_t*>(w->g_ffn);
      o.U = U;
      o.rowsq = rowsq;
    }
    if ((st = launch_gemm(o, P, cnt + L.cnt_off[1], err, s)) != VT_OK) return st;
  }
  if (ffn) {
    if (!attn) {
      hipLaunchKernelGGL(pf::rmsnorm_rows_kernel, dim3(n_tok), dim3(pf::RT), 0, s,
                         static_cast<const uint16_t*>(io->h), static_cast<const uint16_t*>(w->g_ffn),
                         U, static_cast<int>(H), D.rms_eps, cnt, L.ncnt, static_cast<float*>(nullptr),
                         static_cast<int>(d), pos0, D.rope_base);
      if ((st = check("rmsnorm")) != VT_OK) return st;
    }
    // gate/up; epilogue: the RMSNorm's 1 / rms (when the O epilogue left
    // the sums of squares) and M = silu(gate) * up
    pf::GemmArgs a = gemm(2, U, pf::EPI_GU);
    a.b[0] = bsrc(w->wg, w->ld_g, 0, F);
    a.b[1] = bsrc(w->wu, w->ld_u, 0, F);
    a.nb = 2;
    a.interleave = 1;
    a.rowsq = attn ? rowsq : nullptr;
    a.rowsq_tiles = static_cast<int>((H + pf::GBN - 1) / pf::GBN);
    a.Mo = Mb;
    a.F = F;
    a.kpad = std::max(16, (F + 15) / 16 * 16);
    if ((st = launch_gemm(a, P, cnt + L.cnt_off[2], err, s)) != VT_OK) return st;
    // down; epilogue: y = h + p_ffn + peer
    pf::GemmArgs b = gemm(3, Mb, pf::EPI_DOWN);
    b.b[0] = bsrc(w->wd, w->ld_d, 0, gm.N[3]);
    b.nb = 1;
    b.base = static_cast<const uint16_t*>(io->h);
    b.peer = static_cast<const uint16_t*>(io->peer_ffn);
    b.partial = static_cast<uint16_t*>(io->ffn_partial);
    b.out = static_cast<uint16_t*>(io->y);
    if ((st = launch_gemm(b, P, cnt + L.cnt_off[3], err, s)) != VT_OK) return st;
  }
  if (attn) kv->len = pos0 + n_tok;
  return VT_OK;
}
