// Batch-1 decode of one device's shard of a decoder layer on gfx950.
//
// One step (paper Sec. 2.1 decode; Sec. 3.2.1 tensor-parallel shard) runs as
// five phases over a persistent grid of one 512-thread workgroup per CU:
//   0 QKV     RMSNorm(x) * g_attn, then the shard's Wq/Wk/Wv rows (GEMV)
//   1 ATTN    RoPE of q and k, append k and v at slot pos, attention over
//             positions 0..pos split into 32/64-position chunks per KV group,
//             merged by the last chunk to finish (log-sum-exp)
//   2 O       Wo[:, shard heads] * o  -> attn_partial, h = x + partial + peer
//   3 GATEUP  RMSNorm(h) * g_ffn, the shard's Wg/Wu rows, silu(gate) * up
//   4 DOWN    Wd[:, shard cols] * m   -> ffn_partial, y = h + partial + peer
// Decode is bound by streaming the shard's weights from HBM once. Every
// GEMV phase splits its rows evenly over the workgroups; a workgroup's rows
// form one contiguous run of 1 KiB pieces (64 lanes x 16 B) that its eight
// waves split into contiguous sub-runs. Weights do not depend on the
// previous phase, so each wave issues its first 16 pieces before waiting at
// the grid barrier: the barrier's latency overlaps with HBM traffic. Per-row
// sums are reduced in a fixed order (no float atomics), so results are
// bitwise reproducible.
//
// The same kernel also runs one phase per launch (VT_STAGED), with no grid
// barrier; stream order then separates the phases.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <mutex>
#include <vector>

#include "device.hpp"
#include "internal.hpp"

namespace vt {
namespace dec {

constexpr int NT = 512;          // threads per workgroup (8 waves)
constexpr int NW = NT / kWave;   // waves per workgroup
constexpr int PF = 16;           // pieces in flight per wave
constexpr int PRE = 16;          // of which issued before the phase's barrier wait
constexpr int MAX_SLOTS = 4096;  // pieces per workgroup round (one float each)
constexpr int REC = 4;           // attention partial record = head_dim + REC floats
constexpr unsigned kSpinLimit = 1u << 20;  // about a second of polling

enum { PH_QKV = 0, PH_ATTN = 1, PH_O = 2, PH_GATEUP = 3, PH_DOWN = 4 };
// Synchronisation words, each kind in its own 4 KiB-separated spot so that
// the grid barrier's pollers do not share a memory channel with the
// per-head counters of the attention phase. The grid barrier counts
// arrivals on NBAR counters (workgroup b on counter b % NBAR, BAR_STRIDE
// words apart): agent-scope atomics on one word are performed one after
// another, and 256 of them on a single counter made a barrier cost about
// three times as much as on sixteen (measured on MI355X).
constexpr int NBAR = 16, BAR_STRIDE = 32;
enum {
  SW_BAR = 0,
  SW_EXIT = 1024,                        // exit counters, same layout
  SW_EXIT_TOP = SW_EXIT + NBAR * BAR_STRIDE,  // groups whose workgroups have all left
  SW_ERR = 2048,
  SW_GROUP = 3072,
  SW_GROUP_STRIDE = 32
};

struct Params {
  int H, d, nq, nkv, G, ncols, pos, cap, nchunk, cl;
  int p_first;  // first position attended (a sliding window's start, else 0)
  float eps, rope_base;
  const uint16_t *g_attn, *g_ffn;
  // Weight matrices: fp16 values, or block codes (FMT_Q8 / FMT_Q4) with
  // their fp16 block scales; row strides in bytes.
  const uint8_t *wq, *wk, *wv, *wo, *wg, *wu, *wd;
  int64_t ld_q, ld_k, ld_v, ld_o, ld_g, ld_u, ld_d;
  const uint16_t *sq, *sk, *sv, *so, *sg, *su, *sd;
  int64_t lds_q, lds_k, lds_v, lds_o, lds_g, lds_u, lds_d;
  uint16_t *kc, *vc;
  uint32_t kv_bytes;  // bytes of each of kc, vc (n_kv * cap * d * 2)
  const uint16_t *x, *peer_a, *peer_f;
  uint16_t *p_attn, *h, *p_ffn, *y;
  float *qkv, *part, *o, *m;
  float* hbuf;      // h in fp32, shared between the O and FFN phases of one call
  int h_from_ws;    // FFN phases read h from hbuf (1) or from the caller's h (0)
  unsigned* sync;
  int phase_begin, phase_end;
};

// ---------------------------------------------------------------------------
// grid barrier (only between phases of one persistent launch)
// ---------------------------------------------------------------------------
// Data crossing the barrier moves through st_shared / ld_shared only, so
// arrival is: every wave's stores complete, then one relaxed increment of
// the workgroup's counter.
__device__ __forceinline__ void grid_arrive(unsigned* sync) {
  mem_done();
  __syncthreads();
  if (threadIdx.x == 0)
    __hip_atomic_fetch_add(sync + SW_BAR + BAR_STRIDE * (blockIdx.x % NBAR), 1u, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

// Workgroups counting on counter i of NBAR.
__device__ __forceinline__ unsigned bar_group_size(unsigned i) {
  return i < gridDim.x ? (gridDim.x - i + NBAR - 1) / NBAR : 0u;
}

// Wait until every workgroup has arrived ``k`` times: lane i < NBAR of wave
// 0 polls counter i.
__device__ __forceinline__ void grid_wait(unsigned* sync, unsigned k) {
  if (threadIdx.x < NBAR) {
    const unsigned target = k * bar_group_size(threadIdx.x);
    unsigned n = 0;
    while (__hip_atomic_load(sync + SW_BAR + BAR_STRIDE * threadIdx.x, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT) < target) {
      __builtin_amdgcn_s_sleep(2);
      if (++n > kSpinLimit) {  // never expected: report instead of hanging
        sync_or(sync + SW_ERR, 1u);
        break;
      }
    }
  }
  __syncthreads();
}

// At the end of a launch with grid barriers: the last workgroup out (the
// last of the last group to empty) zeroes the barrier and exit counters for
// the next launch.
__device__ __forceinline__ void grid_exit(unsigned* sync) {
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned g = blockIdx.x % NBAR;
    const unsigned old = __hip_atomic_fetch_add(sync + SW_EXIT + BAR_STRIDE * g, 1u, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
    if (old == bar_group_size(g) - 1) {
      const unsigned ngroups = min(gridDim.x, static_cast<unsigned>(NBAR));
      const unsigned top =
          __hip_atomic_fetch_add(sync + SW_EXIT_TOP, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (top == ngroups - 1) {
        for (int i = 0; i < NBAR; ++i) {
          sync_store(sync + SW_BAR + BAR_STRIDE * i, 0u);
          sync_store(sync + SW_EXIT + BAR_STRIDE * i, 0u);
        }
        sync_store(sync + SW_EXIT_TOP, 0u);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// row sources: virtual row index -> (buffer, byte offset of the row). The row
// index is wave-uniform, so the buffer selection stays in scalar registers.
// ---------------------------------------------------------------------------
struct Mat {
  rsrc_t r;      // values or codes
  uint32_t ld;   // row stride in bytes
  rsrc_t s;      // block scales (quantised formats)
  uint32_t lds;  // row stride of the scales in bytes
};

__device__ __forceinline__ Mat make_mat(const uint8_t* w, int64_t ld, int64_t rows, const uint16_t* sc,
                                        int64_t lds) {
  return Mat{make_rsrc(w, static_cast<uint32_t>(rows * ld)), static_cast<uint32_t>(ld),
             make_rsrc(sc, static_cast<uint32_t>(rows * lds)), static_cast<uint32_t>(lds)};
}

// Row r of a row source: the buffer and byte offset of its values / codes
// and of its block scales.
struct RowAt {
  rsrc_t rs, ss;
  uint32_t off, soff;
};

__device__ __forceinline__ RowAt mat_row(const Mat& m, int r) {
  return RowAt{m.r, m.s, static_cast<uint32_t>(r) * m.ld, static_cast<uint32_t>(r) * m.lds};
}

// Every row source also gives the byte offset of a row's segment sg (a
// piece of 1 KiB); only the MoE down projection maps segments elsewhere.
// kSlotTail: the row is several inputs one after the other, each ending in
// a partial segment whose weight columns past col_limit are masked (plain
// rows mask only past K).
__device__ __forceinline__ uint32_t plain_seg(int sg) { return static_cast<uint32_t>(sg) * 1024u; }

struct RowsQKV {
  static constexpr bool kSlotTail = false;
  Mat q, k, v;
  int nqd, nkd;
  __device__ __forceinline__ uint32_t seg_off(int sg) const { return plain_seg(sg); }
  __device__ __forceinline__ RowAt at(int r) const {
    return r < nqd ? mat_row(q, r) : r < nqd + nkd ? mat_row(k, r - nqd) : mat_row(v, r - nqd - nkd);
  }
};

struct RowsOne {
  static constexpr bool kSlotTail = false;
  Mat m;
  __device__ __forceinline__ uint32_t seg_off(int sg) const { return plain_seg(sg); }
  __device__ __forceinline__ RowAt at(int r) const { return mat_row(m, r); }
};

struct RowsPair {  // row 2j -> a[j], row 2j+1 -> b[j]
  static constexpr bool kSlotTail = false;
  Mat a, b;
  __device__ __forceinline__ uint32_t seg_off(int sg) const { return plain_seg(sg); }
  __device__ __forceinline__ RowAt at(int r) const { return (r & 1) ? mat_row(b, r >> 1) : mat_row(a, r >> 1); }
};

// Weight formats of the GEMV phases: fp16 values, or blocks of 32 columns
// with an fp16 scale and INT8 / INT4 codes. A piece is 16 bytes per lane;
// EPL is the number of columns a lane covers in it.
enum { FMT_F16 = 0, FMT_Q8 = 1, FMT_Q4 = 2 };
template <int F>
struct Fmt {
  static constexpr int EPL = F == FMT_F16 ? 8 : F == FMT_Q8 ? 16 : 32;
  static constexpr int SEGC = 64 * EPL;  // columns per piece
};

__host__ __device__ __forceinline__ int seg_cols(int fmt) { return fmt == FMT_F16 ? 512 : fmt == FMT_Q8 ? 1024 : 2048; }

// Zero the fp16 weights of columns >= K in a lane's 8-column chunk starting
// at ``col`` (row padding may hold anything).
__device__ __forceinline__ u32x4 mask_tail(u32x4 w, int col, int K) {
  const int v = K - col;
  w.x = v >= 2 ? w.x : (v >= 1 ? (w.x & 0xFFFFu) : 0u);
  w.y = v >= 4 ? w.y : (v >= 3 ? (w.y & 0xFFFFu) : 0u);
  w.z = v >= 6 ? w.z : (v >= 5 ? (w.z & 0xFFFFu) : 0u);
  w.w = v >= 8 ? w.w : (v >= 7 ? (w.w & 0xFFFFu) : 0u);
  return w;
}

// acc + sum of the 8 products of fp16 weights w and fp16 inputs x (fp32
// accumulate, two products per instruction). The halves are taken with
// vector shuffles of the whole 16 bytes: bit-casting single ext-vector
// elements (w.y, ...) makes this compiler reuse element 0 for all four.
__device__ __forceinline__ float dot8(const u32x4 w, const u32x4 x, float acc) {
  const f16x8 a = __builtin_bit_cast(f16x8, w), b = __builtin_bit_cast(f16x8, x);
  acc = __builtin_amdgcn_fdot2(__builtin_shufflevector(a, a, 0, 1), __builtin_shufflevector(b, b, 0, 1),
                               acc, false);
  acc = __builtin_amdgcn_fdot2(__builtin_shufflevector(a, a, 2, 3), __builtin_shufflevector(b, b, 2, 3),
                               acc, false);
  acc = __builtin_amdgcn_fdot2(__builtin_shufflevector(a, a, 4, 5), __builtin_shufflevector(b, b, 4, 5),
                               acc, false);
  acc = __builtin_amdgcn_fdot2(__builtin_shufflevector(a, a, 6, 7), __builtin_shufflevector(b, b, 6, 7),
                               acc, false);
  return acc;
}

// One GEMV phase over ``units`` output units of U virtual rows of K columns.
// A row is split into segments of 512 columns; a piece is one segment of
// one row (64 lanes x 16 B). Wave 0 is the control wave: it holds no weight
// loads, so it can wait at the grid barrier and stage the phase's input
// while the other (streaming) waves' first PF loads are in flight; memory
// ordering is in-order per wave, so a wave holding loads could not see the
// barrier flip before they land. The workgroup's rows form a contiguous run
// of pieces that the streaming waves split into contiguous sub-runs; each
// streams its sub-run through a ring of PF loads, accumulates a row's
// segments in each lane and reduces across the wave at the row's end (or
// where its sub-run ends), writing the sum to slots[piece]. ``stage`` (run
// by wave 0 alone) writes the input as fp16 to xs16[0, nseg*512), zero past
// K. ``epi(unit, sums)`` gets each unit's U row sums, added in piece order.
// q / n for 0 <= q < 2^24 / n, with rcp = floor(2^24 / n) + 1: a scalar
// multiply and shift (exact in that range; pieces per round stay < 2^13).
__device__ __forceinline__ int div_rcp(int q, uint32_t rcp) {
  return static_cast<int>((static_cast<uint64_t>(static_cast<uint32_t>(q)) * rcp) >> 24);
}

// Codes to fp16 pairs. A byte u placed under the high byte 0x64 is the fp16
// number 1024 + u exactly; v_perm_b32 builds two such halves from bytes
// ``i`` and ``j`` of ``src`` (selector bytes 0-3 pick from its second
// operand, 4 from the first: 0x64), then the offset (1024 plus the code's
// bias) is subtracted exactly.
__device__ __forceinline__ f16x2 code_pair(uint32_t src, uint32_t sel, _Float16 off) {
  const uint32_t w = __builtin_amdgcn_perm(0x64646464u, src, sel);
  return __builtin_bit_cast(f16x2, w) - f16x2{off, off};
}
constexpr uint32_t kSel01 = 0x04010400u;  // bytes 0 and 1 -> (1024 + b0, 1024 + b1)
constexpr uint32_t kSel23 = 0x04030402u;  // bytes 2 and 3

__device__ __forceinline__ float dot2h(f16x2 a, uint32_t x, float acc) {
  return __builtin_amdgcn_fdot2(a, __builtin_bit_cast(f16x2, x), acc, false);
}

// Sum of 16 INT8 codes (two's complement, column order) times 16 fp16
// inputs (xa: columns 0-7, xb: 8-15).
__device__ __forceinline__ float dot_q8(const u32x4 w, const u32x4 xa, const u32x4 xb) {
  const uint32_t wv[4] = {w.x, w.y, w.z, w.w};
  const uint32_t xv[8] = {xa.x, xa.y, xa.z, xa.w, xb.x, xb.y, xb.z, xb.w};
  float acc = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t t = wv[j] ^ 0x80808080u;  // code + 128 in each byte
    acc = dot2h(code_pair(t, kSel01, 1152), xv[2 * j], acc);
    acc = dot2h(code_pair(t, kSel23, 1152), xv[2 * j + 1], acc);
  }
  return acc;
}

// Sum of 32 INT4 codes (offset-binary nibbles; in each 32-bit word the low
// nibbles are columns 0-3 and the high nibbles columns 4-7 of its group of
// 8) times 32 fp16 inputs x[0..3] (8 columns each).
__device__ __forceinline__ float dot_q4(const u32x4 w, const u32x4 (&x)[4]) {
  const uint32_t wv[4] = {w.x, w.y, w.z, w.w};
  float acc = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t lo = wv[j] & 0x0F0F0F0Fu, hi = (wv[j] >> 4) & 0x0F0F0F0Fu;
    acc = dot2h(code_pair(lo, kSel01, 1032), x[j].x, acc);
    acc = dot2h(code_pair(lo, kSel23, 1032), x[j].y, acc);
    acc = dot2h(code_pair(hi, kSel01, 1032), x[j].z, acc);
    acc = dot2h(code_pair(hi, kSel23, 1032), x[j].w, acc);
  }
  return acc;
}

// Block scales of a quantised format are staged per round in LDS (the
// rows' scale vectors, up to SC_ROW_WORDS 32-bit words a row per lane):
// a 2-byte load per piece and lane would double the memory instructions of
// the weight stream, and the CU's memory pipeline is limited by those.
constexpr int SC_ROWS = 32;       // scale rows per round (a workgroup)
constexpr int SC_ROW_WORDS = 4;   // 32-bit words per lane and row: up to 512 blocks (K <= 16384)
constexpr int SC_LDS_HALFS = SC_ROWS * SC_ROW_WORDS * 2 * kWave;  // 32 rows x 512 scales
// (a phase is compiled for 1, 2 and 4 words per lane and row, and runs the
// smallest that holds its rows' blocks: every load, even one that reads
// past its buffer, costs the memory pipeline an instruction)
constexpr int SC_PER_WAVE = (SC_ROWS + NW - 1) / NW;

template <int U, int F, int SCW, class Rows, class Stage, class Epi>
__device__ __forceinline__ void gemv_impl(const Rows& rows, int units, int K, const uint16_t* xs16,
                                          float* slots, uint16_t* scl, Stage stage, Epi epi) {
  constexpr int EPL = Fmt<F>::EPL, SEGC = Fmt<F>::SEGC;
  constexpr bool QUANT = F != FMT_F16;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = threadIdx.x % kWave;
  const int u0 = static_cast<int>(static_cast<int64_t>(units) * blockIdx.x / gridDim.x);
  const int u1 = static_cast<int>(static_cast<int64_t>(units) * (blockIdx.x + 1) / gridDim.x);
  const int nseg = max(1, (K + SEGC - 1) / SEGC);
  const uint32_t rcp = (1u << 24) / static_cast<uint32_t>(nseg) + 1u;
  const int tail = K - (nseg - 1) * SEGC;  // columns in a row's last segment
  const uint32_t lane16 = static_cast<uint32_t>(lane) * 16u;
  const bool lane_in_tail = lane * EPL < tail;
  // scale rows in LDS: nbp fp16 per row (the row's blocks, rounded up to
  // whole 32-bit words of every lane's share)
  const int nb = (K + 31) / 32;
  const int sc_words = (nb + 2 * kWave - 1) / (2 * kWave);  // 32-bit loads per lane and row
  const int nbp = sc_words * 2 * kWave;
  int upr = max(1, MAX_SLOTS / (U * nseg));
  if constexpr (QUANT) upr = max(1, min(upr, SC_ROWS / U));
  // Load piece p (row p / nseg, segment p % nseg of this round) into a
  // register quad; p >= q1 (past the wave's run) reads zero without memory
  // traffic. kOOB is OR-ed in arithmetically: a select here can become a
  // branch around the load, and the branch a full wait for every load in
  // flight.
  auto issue = [&](int row0, int p, int q1) -> u32x4 {
    const int lr = div_rcp(p, rcp);
    const int sg = p - lr * nseg;
    const RowAt ra = rows.at(row0 + lr);
    const uint32_t base = __builtin_amdgcn_readfirstlane(ra.off + rows.seg_off(sg));
    const bool ok = (p < q1) && (sg != nseg - 1 || lane_in_tail);
    const uint32_t oob = static_cast<uint32_t>(!ok) << 31;
    return __builtin_amdgcn_raw_buffer_load_b128(ra.rs, (base + lane16) | oob, 0, 0);
  };
  bool staged = false;
  int ua = u0;
  do {
    const int ub = min(u1, ua + upr);
    const int np = K > 0 ? (ub - ua) * U * nseg : 0;
    const int q0 = __builtin_amdgcn_readfirstlane(static_cast<int>(static_cast<int64_t>(np) * wave / NW));
    const int q1 = __builtin_amdgcn_readfirstlane(static_cast<int>(static_cast<int64_t>(np) * (wave + 1) / NW));
    const int row0 = ua * U;
    for (int i = threadIdx.x; i < np; i += NT) slots[i] = 0.f;
    u32x4 buf[PF];
    // A few pieces go out before the barrier wait: they cover its latency
    // without queueing so much traffic that the staging loads behind them
    // stall. The rest of the ring follows once the input is staged.
    // in groups of 4, only as far as the run goes (a load past it still
    // costs the memory pipeline an instruction)
#pragma unroll
    for (int g = 0; g < PRE / 4; ++g) {
      if (g == 0 || q0 + 4 * g < q1) {
#pragma unroll
        for (int i = 4 * g; i < 4 * g + 4; ++i) buf[i] = issue(row0, q0 + i, q1);
      }
    }
    // The round's scale rows (row vr on wave vr % NW); they are written to
    // LDS once the input is staged, when they have long landed.
    uint32_t sreg[QUANT ? SC_PER_WAVE : 1][SCW];
    if constexpr (QUANT) {
      const int nr = K > 0 ? (ub - ua) * U : 0;
#pragma unroll
      for (int k = 0; k < SC_PER_WAVE; ++k) {
        const int vr = wave + k * NW;
        const RowAt ra = rows.at(row0 + min(vr, max(nr - 1, 0)));
#pragma unroll
        for (int w = 0; w < SCW; ++w) {
          const int idx = w * kWave + lane;  // word of the row: scales 2 idx, 2 idx + 1
          const uint32_t oob = static_cast<uint32_t>(!(vr < nr && 2 * idx < nb)) << 31;
          const uint32_t v =
              __builtin_amdgcn_raw_buffer_load_b32(ra.ss, (ra.soff + static_cast<uint32_t>(idx) * 4u) | oob, 0, 0);
          // past the row's last block the scale is 0 (the codes there are 0
          // or unread, and 0 * 0 must stay 0 whatever the padding holds)
          sreg[k][w] = 2 * idx + 1 < nb ? v : (v & 0xFFFFu);
        }
      }
    }
    if (!staged) {
      stage();  // all threads; ends with a workgroup barrier
      staged = true;
    } else {
      __syncthreads();
    }
#pragma unroll
    for (int i = PRE; i < PF; ++i) buf[i] = issue(row0, q0 + i, q1);
    // The scale rows go to LDS once the input is staged: their loads left
    // first, so they have landed by now and the wait costs nothing.
    if constexpr (QUANT) {  // scale rows to LDS: row vr at scl + vr * nbp
      const int nr = K > 0 ? (ub - ua) * U : 0;
#pragma unroll
      for (int k = 0; k < SC_PER_WAVE; ++k) {
        const int vr = wave + k * NW;
        if (vr < nr) {
          uint32_t* dst = reinterpret_cast<uint32_t*>(scl + vr * nbp);
#pragma unroll
          for (int w = 0; w < SCW; ++w)
            if (w < sc_words) dst[w * kWave + lane] = sreg[k][w];
        }
      }
      lds_barrier();
    }
    // The wave's run in trips of PF pieces; every trip but the last reloads
    // the ring (a load past the run reads zero but still costs the memory
    // pipeline an instruction).
    float acc = 0.f;
    const int ntrip = (q1 - q0 + PF - 1) / PF;
    auto trip = [&](int base, bool reload) {
#pragma unroll
      for (int i = 0; i < PF; ++i) {
        const int q = base + i;
        if (q < q1) {
          const int lr = div_rcp(q, rcp);
          const int cs = q - lr * nseg;
          const int col = cs * SEGC + lane * EPL;
          const u32x4* xp = reinterpret_cast<const u32x4*>(xs16 + col);
          if constexpr (F == FMT_F16) {
            u32x4 w = buf[i];
            if constexpr (Rows::kSlotTail)
              w = mask_tail(w, col, rows.col_limit(cs));
            else if (cs == nseg - 1 && tail < SEGC)
              w = mask_tail(w, col, K);
            acc = dot8(w, xp[0], acc);
          } else {
            // codes past K are zero by the format, and so is the input
            const float sc = h2f(scl[lr * nbp + col / 32]);
            if constexpr (F == FMT_Q8) {
              acc = fmaf(sc, dot_q8(buf[i], xp[0], xp[1]), acc);
            } else {
              const u32x4 xq[4] = {xp[0], xp[1], xp[2], xp[3]};
              acc = fmaf(sc, dot_q4(buf[i], xq), acc);
            }
          }
          if (cs == nseg - 1 || q == q1 - 1) {
            const float t = wave_sum(acc);
            if (lane == 0) slots[q] = t;
            acc = 0.f;
          }
        }
        if (reload) buf[i] = issue(row0, q + PF, q1);
      }
    };
    for (int tr = 0; tr + 1 < ntrip; ++tr) trip(q0 + tr * PF, true);
    if (ntrip > 0) trip(q0 + (ntrip - 1) * PF, false);
    lds_barrier();  // every slot written
    for (int lu = threadIdx.x; lu < ub - ua; lu += NT) {
      float v[U];
#pragma unroll
      for (int j = 0; j < U; ++j) {
        float a = 0.f;
        if (K > 0) {
          const float* sl = slots + (lu * U + j) * nseg;
          for (int s = 0; s < nseg; ++s) a += sl[s];
        }
        v[j] = a;
      }
      epi(ua + lu, v);
    }
    lds_barrier();  // slots, scales and xs free for reuse
    ua = ub;
  } while (ua < u1);
}

template <int U, int F, class Rows, class Stage, class Epi>
__device__ __forceinline__ void gemv_phase(const Rows& rows, int units, int K, const uint16_t* xs16,
                                           float* slots, uint16_t* scl, Stage stage, Epi epi) {
  if constexpr (F == FMT_F16) {
    gemv_impl<U, F, 1>(rows, units, K, xs16, slots, scl, stage, epi);
  } else {
    const int words = ((K + 31) / 32 + 2 * kWave - 1) / (2 * kWave);  // per lane and scale row
    if (words <= 1)
      gemv_impl<U, F, 1>(rows, units, K, xs16, slots, scl, stage, epi);
    else if (words <= 2)
      gemv_impl<U, F, 2>(rows, units, K, xs16, slots, scl, stage, epi);
    else
      gemv_impl<U, F, SC_ROW_WORDS>(rows, units, K, xs16, slots, scl, stage, epi);
  }
}

// ---------------------------------------------------------------------------
// staging of a GEMV phase's input vector into LDS as fp16 (all threads; each
// ends with a workgroup barrier)
// ---------------------------------------------------------------------------
// xs[k] = fp16(v[k] * rstd * g[k]), rstd = 1 / sqrt(mean(v^2) + eps), for a
// caller-provided fp16 vector v (n a multiple of 8, n <= 8 * 4 * NT); zero
// for n <= k < npad.
__device__ __forceinline__ void stage_rmsnorm_h(const uint16_t* v, const uint16_t* g, int n, int npad,
                                                float eps, uint16_t* xs, float* red) {
  constexpr int MAXC = 4;
  const int nch = n / 8;
  const rsrc_t rv = make_rsrc(v, static_cast<uint32_t>(n) * 2u);
  const rsrc_t rg = make_rsrc(g, static_cast<uint32_t>(n) * 2u);
  u32x4 xv[MAXC], gv[MAXC];
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {  // chunks past n read as zero
    const uint32_t off = static_cast<uint32_t>(threadIdx.x + c * NT) * 16u;
    xv[c] = buf_load16(rv, off);
    gv[c] = buf_load16(rg, off);
  }
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    float f[8];
    unpack8(xv[c], f);
#pragma unroll
    for (int e = 0; e < 8; ++e) ss = fmaf(f[e], f[e], ss);
  }
  ss = block_sum<NT>(ss, red);
  const float rstd = 1.0f / sqrtf(ss / static_cast<float>(n) + eps);
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    const int k8 = threadIdx.x + c * NT;
    if (k8 < nch) {
      float f[8], gf[8];
      unpack8(xv[c], f);
      unpack8(gv[c], gf);
#pragma unroll
      for (int e = 0; e < 8; ++e) xs[k8 * 8 + e] = f2h(f[e] * rstd * gf[e]);
    }
  }
  for (int k = n + threadIdx.x; k < npad; k += NT) xs[k] = 0;
  __syncthreads();
}

// The same for an fp32 vector written by other workgroups of this launch
// (n a multiple of 8), each value first rounded to fp16: the value the
// caller's fp16 h would carry.
__device__ __forceinline__ void stage_rmsnorm_f(const float* v, const uint16_t* g, int n, int npad,
                                                float eps, uint16_t* xs, float* red) {
  constexpr int MAXP = 16;  // float pairs held per thread
  const int npair = n / 2;
  float a[MAXP] = {}, b[MAXP] = {};
  uint32_t gw[MAXP] = {};  // the two fp16 gains of each pair (zero past n)
  // Unconditional buffer loads (coherent for the values): pairs past n read
  // zero without memory traffic (a guarded load would get a branch and a
  // full wait each). Each pair's value and gain loads go out together; that
  // order measured faster than all values first, then all gains.
  const rsrc_t rv = make_rsrc(v, static_cast<uint32_t>(npair) * 8u);
  const rsrc_t rg = make_rsrc(g, static_cast<uint32_t>(n) * 2u);
#pragma unroll
  for (int u = 0; u < MAXP; ++u) {
    buf_ld_shared2(rv, static_cast<uint32_t>(threadIdx.x + u * NT) * 8u, a[u], b[u]);
    gw[u] = __builtin_amdgcn_raw_buffer_load_b32(rg, static_cast<uint32_t>(threadIdx.x + u * NT) * 4u, 0, 0);
  }
  float ss = 0.f;
#pragma unroll
  for (int u = 0; u < MAXP; ++u) {
    const bool ok = static_cast<int>(threadIdx.x) + u * NT < npair;
    a[u] = ok ? round_h(a[u]) : 0.f;
    b[u] = ok ? round_h(b[u]) : 0.f;
    ss = fmaf(a[u], a[u], fmaf(b[u], b[u], ss));
  }
  ss = block_sum<NT>(ss, red);
  const float rstd = 1.0f / sqrtf(ss / static_cast<float>(n) + eps);
#pragma unroll
  for (int u = 0; u < MAXP; ++u) {
    const int i = threadIdx.x + u * NT;
    if (i < npair) {
      float g0, g1;
      unpack2(gw[u], g0, g1);
      xs[2 * i] = f2h(a[u] * rstd * g0);
      xs[2 * i + 1] = f2h(b[u] * rstd * g1);
    }
  }
  for (int k = n + threadIdx.x; k < npad; k += NT) xs[k] = 0;
  __syncthreads();
}

// xs[k] = fp16(v[k]) for an fp32 vector written by other workgroups of this
// launch (its buffer holds an even number of floats); zero for n <= k < npad.
__device__ __forceinline__ void stage_copy_f(const float* v, int n, int npad, uint16_t* xs) {
  constexpr int MAXP = 16;
  const int npair = (n + 1) / 2;
  const rsrc_t rv = make_rsrc(v, static_cast<uint32_t>(npair) * 8u);
  for (int c0 = 0; c0 < npair; c0 += MAXP * NT) {
    float a[MAXP] = {}, b[MAXP] = {};
#pragma unroll
    for (int u = 0; u < MAXP; ++u)  // unconditional, zero past the end (see stage_rmsnorm_f)
      buf_ld_shared2(rv, static_cast<uint32_t>(c0 + threadIdx.x + u * NT) * 8u, a[u], b[u]);
#pragma unroll
    for (int u = 0; u < MAXP; ++u) {
      const int i = c0 + threadIdx.x + u * NT;
      if (i < npair) {
        xs[2 * i] = f2h(a[u]);
        xs[2 * i + 1] = 2 * i + 1 < n ? f2h(b[u]) : 0;
      }
    }
  }
  for (int k = 2 * npair + threadIdx.x; k < npad; k += NT) xs[k] = 0;
  __syncthreads();
}

// K rounded up to whole pieces of the format's segment.
__host__ __device__ __forceinline__ int padded(int K, int fmt) {
  const int sc = seg_cols(fmt);
  return ((K + sc - 1) / sc) * sc;
}

// ---------------------------------------------------------------------------
// phase 1: attention
//
// Work item = (query head j, chunk of CL consecutive positions). A thread
// holds 8 of the d dimensions of one position per pass (d/8 threads per
// position, PPP positions per pass, CL = passes * PPP). The chunk's keys and
// values do not depend on phase 0, so they are loaded into registers before
// the grid barrier. Items of the G query heads that share a KV head and a
// chunk are placed on workgroups with equal index mod 8, i.e. on one XCD, so
// the group reads each K/V tile from HBM once and from that XCD's L2 after.
// Each item writes (unnormalised sum of p*V, running max m, sum l); the last
// item of head j to finish merges the head's chunks by log-sum-exp.
// ---------------------------------------------------------------------------
constexpr int MAXPASS = 8;

__host__ __device__ __forceinline__ int attn_ppp(int d) { return NT / (d / 8); }

__host__ __device__ __forceinline__ int attn_lds_floats(int d, int nchunk) {
  const int ppp = attn_ppp(d);
  return d + MAXPASS * ppp + ppp * d + 2 * d + 2 * nchunk + 4;
}

__device__ __forceinline__ void phase_attn(const Params& P, float* lds, bool wait, unsigned nbar) {
  const int d = P.d, G = P.G, CL = P.cl;
  const int TPP = d / 8, PPP = NT / TPP, NPASS = CL / PPP;
  const int t = threadIdx.x, wave = t / kWave, lane = t % kWave;
  const int pl = t / TPP;             // position within a pass
  const int dc = (t % TPP) * 8;       // first of this thread's 8 dimensions
  const int RW = d + REC;             // floats per partial record
  const int units = P.nkv * P.nchunk; // (KV head, chunk) pairs
  const int ids = ((units + 7) / 8) * 8 * G;
  const float scale = 1.0f / sqrtf(static_cast<float>(d));
  // LDS (floats): qs[d] | S[MAXPASS*PPP] | R[PPP*d] | kn[d] | vn[d] | W[2*nchunk] | flag
  float* qs = lds;
  float* S = qs + d;
  float* R = S + MAXPASS * PPP;
  float* kn = R + PPP * d;
  float* vn = kn + d;
  float* W = vn + d;
  int* flag = reinterpret_cast<int*>(W + 2 * P.nchunk);
  const rsrc_t rk = make_rsrc(P.kc, P.kv_bytes), rv = make_rsrc(P.vc, P.kv_bytes);

  bool waited = false;
  for (int id = blockIdx.x;; id += gridDim.x) {
    const int r8 = id % 8;
    const int jj = (id / 8) % G;
    const int u = (id / (8 * G)) * 8 + r8;
    const bool valid = id < ids && u < units;
    const int g = valid ? u / P.nchunk : 0;
    const int c = valid ? u - g * P.nchunk : 0;
    const int j = g * G + jj;                 // shard-local query head
    const int p0 = P.p_first + c * CL;
    u32x4 kr[MAXPASS] = {}, vr[MAXPASS] = {};
#pragma unroll
    for (int ps = 0; ps < MAXPASS; ++ps) {
      if (ps == 0 || ps < NPASS) {  // passes of the chunk only (uniform)
        const int p = p0 + ps * PPP + pl;
        const bool ok = valid && p < P.pos;
        const uint32_t off =
            ok ? static_cast<uint32_t>(((static_cast<int64_t>(g) * P.cap + p) * d + dc) * 2) : kOOB;
        kr[ps] = buf_load16(rk, off);
        vr[ps] = buf_load16(rv, off);
      }
    }
    // rotation of pair t at the new position (independent of phase 0)
    const int half = d / 2;
    float c0 = 1.f, s0 = 0.f;
    if (t < half) rope_angle(P.pos, t, d, P.rope_base, c0, s0);
    if (!waited) {
      if (wait) grid_wait(P.sync, nbar);
      waited = true;
    }
    if (id >= ids) break;
    if (!valid) continue;

    // rotated, pre-scaled query of head j; the new token's key and value.
    // Coherent loads are issued unconditionally with clamped indices (a
    // guarded one gets a branch and a full wait of its own).
    const int tp = min(t, half - 1);       // this thread's rotation pair
    const int tv = min(max(t - half, 0), d - 1);
    const float* q = P.qkv + static_cast<int64_t>(j) * d;
    const float* kq = P.qkv + static_cast<int64_t>(P.nq + g) * d;
    const float* vq = P.qkv + static_cast<int64_t>(P.nq + P.nkv + g) * d;
    float qa, qb, ka, kb;
    ld_shared2(q + 2 * tp, qa, qb);
    ld_shared2(kq + 2 * tp, ka, kb);
    const float vv = ld_shared(vq + tv);
    if (t < half) {
      qs[2 * t] = (qa * c0 - qb * s0) * scale;
      qs[2 * t + 1] = (qa * s0 + qb * c0) * scale;
    }
    const bool has_new = P.pos >= p0 && P.pos < p0 + CL;
    if (has_new) {  // the new token's key (rotated) and value, rounded as stored
      const int64_t slot = (static_cast<int64_t>(g) * P.cap + P.pos) * d;
      const bool writer = jj == 0;  // one item per KV head appends to the cache
      if (t < half) {
        const float a = ka, b = kb;
        const uint16_t k0 = f2h(a * c0 - b * s0), k1 = f2h(a * s0 + b * c0);
        kn[2 * t] = h2f(k0);
        kn[2 * t + 1] = h2f(k1);
        if (writer) {
          P.kc[slot + 2 * t] = k0;
          P.kc[slot + 2 * t + 1] = k1;
        }
      } else if (t < half + d) {
        const int i = t - half;
        const uint16_t v0 = f2h(vv);
        vn[i] = h2f(v0);
        if (writer) P.vc[slot + i] = v0;
      }
    }
    __syncthreads();

    // scores
#pragma unroll
    for (int ps = 0; ps < MAXPASS; ++ps) {
      if (ps < NPASS) {
        const int p = p0 + ps * PPP + pl;
        float kf[8];
        unpack8(kr[ps], kf);
        if (p == P.pos) {
#pragma unroll
          for (int e = 0; e < 8; ++e) kf[e] = kn[dc + e];
        }
        float sc = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) sc = fmaf(qs[dc + e], kf[e], sc);
        sc = group_sum(sc, TPP);
        if ((t % TPP) == 0) S[ps * PPP + pl] = p <= P.pos ? sc : -INFINITY;
      }
    }
    __syncthreads();
    float* rec = P.part + (static_cast<int64_t>(j) * P.nchunk + c) * RW;
    if (wave == 0) {  // softmax statistics of the chunk
      float mx = -INFINITY;
      for (int q = lane; q < CL; q += kWave) mx = fmaxf(mx, S[q]);
      mx = wave_max(mx);
      float l = 0.f;
      for (int q = lane; q < CL; q += kWave) {
        const float e = S[q] == -INFINITY ? 0.f : __expf(S[q] - mx);
        S[q] = e;
        l += e;
      }
      l = wave_sum(l);
      if (lane == 0) {
        st_shared(rec + d, mx);
        st_shared(rec + d + 1, l);
      }
    }
    __syncthreads();
    // unnormalised sum of weights * values over the chunk
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ps = 0; ps < MAXPASS; ++ps) {
      if (ps < NPASS) {
        const int p = p0 + ps * PPP + pl;
        const float e = S[ps * PPP + pl];
        float vf[8];
        unpack8(vr[ps], vf);
        if (p == P.pos) {
#pragma unroll
          for (int x = 0; x < 8; ++x) vf[x] = vn[dc + x];
        }
#pragma unroll
        for (int x = 0; x < 8; ++x) acc[x] = fmaf(e, vf[x], acc[x]);
      }
    }
#pragma unroll
    for (int x = 0; x < 8; ++x) R[pl * d + dc + x] = acc[x];
    __syncthreads();
    for (int dd = t; dd < d; dd += NT) {
      float a = 0.f;
      for (int q = 0; q < PPP; ++q) a += R[q * d + dd];
      st_shared(rec + dd, a);
    }

    // the last chunk of head j to finish merges the head's chunks
    mem_done();
    __syncthreads();
    if (t == 0) {
      const unsigned old = __hip_atomic_fetch_add(P.sync + SW_GROUP + j * SW_GROUP_STRIDE, 1u, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
      *flag = (old == static_cast<unsigned>(P.nchunk - 1));
    }
    __syncthreads();
    if (*flag) {
      // Thread (grp, dd) takes chunks grp, grp + ngrp, ...: it loads their
      // (m, l, value[dd]) in batches of 16 (one round trip each) and keeps a
      // running (max, sum l, sum value) under the log-sum-exp rescaling; the
      // ngrp partial triples of each dd are then merged in a fixed order.
      const rsrc_t rj = make_rsrc(P.part + static_cast<int64_t>(j) * P.nchunk * RW,
                                  static_cast<uint32_t>(P.nchunk * RW) * 4u);
      const int ngrp = NT / d, grp = t / d, dd = t % d;
      float M = -INFINITY, Ls = 0.f, A = 0.f;
      for (int c0 = grp; grp < ngrp && c0 < P.nchunk; c0 += 16 * ngrp) {
        float mv[16], lv[16], ov[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) {  // unconditional; chunks past the last read zero
          const int cc = c0 + u * ngrp;
          const uint32_t rec = cc < P.nchunk ? static_cast<uint32_t>(cc * RW) * 4u : kOOB;
          buf_ld_shared2(rj, rec == kOOB ? kOOB : rec + d * 4u, mv[u], lv[u]);
          ov[u] = buf_ld_shared(rj, rec == kOOB ? kOOB : rec + dd * 4u);
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          if (c0 + u * ngrp >= P.nchunk) {
            mv[u] = -INFINITY;
            lv[u] = 0.f;
            ov[u] = 0.f;
          }
        }
        float bm = M;
#pragma unroll
        for (int u = 0; u < 16; ++u) bm = fmaxf(bm, mv[u]);
        const float r = M == -INFINITY ? 0.f : __expf(M - bm);
        Ls *= r;
        A *= r;
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          const float w = mv[u] == -INFINITY ? 0.f : __expf(mv[u] - bm);
          Ls = fmaf(lv[u], w, Ls);
          A = fmaf(ov[u], w, A);
        }
        M = bm;
      }
      if (grp < ngrp) {
        R[(3 * grp + 0) * d + dd] = M;
        R[(3 * grp + 1) * d + dd] = Ls;
        R[(3 * grp + 2) * d + dd] = A;
      }
      __syncthreads();
      if (t < d) {
        float Mx = -INFINITY;
        for (int q = 0; q < ngrp; ++q) Mx = fmaxf(Mx, R[(3 * q) * d + t]);
        float Lt = 0.f, At = 0.f;
        for (int q = 0; q < ngrp; ++q) {
          const float mq = R[(3 * q) * d + t];
          const float w = mq == -INFINITY ? 0.f : __expf(mq - Mx);
          Lt = fmaf(R[(3 * q + 1) * d + t], w, Lt);
          At = fmaf(R[(3 * q + 2) * d + t], w, At);
        }
        st_shared(P.o + static_cast<int64_t>(j) * d + t, At / Lt);
      }
      if (t == 0) sync_store(P.sync + SW_GROUP + j * SW_GROUP_STRIDE, 0u);
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// the kernel
// ---------------------------------------------------------------------------
// One phase; ``wait``: a grid barrier is in front of it, the ``nbar``-th of
// the launch.
template <int PH, int F>
__device__ __forceinline__ void run_phase(const Params& P, float* lds, uint16_t* xs, float* slots,
                                          float* red, bool wait, unsigned nbar) {
  uint16_t* scl = reinterpret_cast<uint16_t*>(red + 16);  // block scales (quantised formats)
  if constexpr (PH == PH_QKV) {
    RowsQKV rows{make_mat(P.wq, P.ld_q, P.nq * P.d, P.sq, P.lds_q),
                 make_mat(P.wk, P.ld_k, P.nkv * P.d, P.sk, P.lds_k),
                 make_mat(P.wv, P.ld_v, P.nkv * P.d, P.sv, P.lds_v), P.nq * P.d, P.nkv * P.d};
    gemv_phase<1, F>(
        rows, (P.nq + 2 * P.nkv) * P.d, P.H, xs, slots, scl,
        [&]() { stage_rmsnorm_h(P.x, P.g_attn, P.H, padded(P.H, F), P.eps, xs, red); },
        [&](int r, const float* v) { st_shared(P.qkv + r, v[0]); });
  } else if constexpr (PH == PH_ATTN) {
    phase_attn(P, lds, wait, nbar);
  } else if constexpr (PH == PH_O) {
    RowsOne rows{make_mat(P.wo, P.ld_o, P.H, P.so, P.lds_o)};
    const int K = P.nq * P.d;
    gemv_phase<1, F>(
        rows, P.H, K, xs, slots, scl,
        [&]() {
          if (wait) grid_wait(P.sync, nbar);
          stage_copy_f(P.o, K, padded(K, F), xs);
        },
        [&](int r, const float* v) {
          const float pa = v[0];
          P.p_attn[r] = f2h(pa);
          const float hv = h2f(P.x[r]) + pa + (P.peer_a ? h2f(P.peer_a[r]) : 0.f);
          P.h[r] = f2h(hv);
          st_shared(P.hbuf + r, hv);
        });
  } else if constexpr (PH == PH_GATEUP) {
    RowsPair rows{make_mat(P.wg, P.ld_g, P.ncols, P.sg, P.lds_g),
                  make_mat(P.wu, P.ld_u, P.ncols, P.su, P.lds_u)};
    gemv_phase<2, F>(
        rows, P.ncols, P.H, xs, slots, scl,
        [&]() {
          if (wait) grid_wait(P.sync, nbar);
          if (P.h_from_ws)
            stage_rmsnorm_f(P.hbuf, P.g_ffn, P.H, padded(P.H, F), P.eps, xs, red);
          else
            stage_rmsnorm_h(P.h, P.g_ffn, P.H, padded(P.H, F), P.eps, xs, red);
        },
        [&](int j, const float* v) {
          const float gt = v[0], up = v[1];
          st_shared(P.m + j, gt / (1.0f + __expf(-gt)) * up);
        });
  } else {
    RowsOne rows{make_mat(P.wd, P.ld_d, P.H, P.sd, P.lds_d)};
    const int K = P.ncols;
    gemv_phase<1, F>(
        rows, P.H, K, xs, slots, scl,
        [&]() {
          if (wait) grid_wait(P.sync, nbar);
          stage_copy_f(P.m, K, padded(K, F), xs);
        },
        [&](int r, const float* v) {
          const float pf = v[0];
          P.p_ffn[r] = f2h(pf);
          if (P.y) {
            const float hr = P.h_from_ws ? round_h(ld_shared(P.hbuf + r)) : h2f(P.h[r]);
            P.y[r] = f2h(hr + pf + (P.peer_f ? h2f(P.peer_f[r]) : 0.f));
          }
        });
  }
}

template <int PH, int PE, int PB, int F>
__device__ __forceinline__ void run_phases(const Params& P, float* lds, uint16_t* xs, float* slots,
                                           float* red) {
  run_phase<PH, F>(P, lds, xs, slots, red, PH > PB, static_cast<unsigned>(PH - PB));
  if constexpr (PH < PE) {
    grid_arrive(P.sync);
    run_phases<PH + 1, PE, PB, F>(P, lds, xs, slots, red);
  }
}

// Phases PB..PE of one decode step. PB < PE needs every workgroup resident
// (one per CU): grid barriers separate the phases.
template <int PB, int PE, int F>
__global__ void __launch_bounds__(NT) decode_kernel(Params P) {
  extern __shared__ float lds[];
  // LDS: xs / attention scratch (aliased) | slots[MAX_SLOTS] | red[16] |
  // block scales (quantised formats)
  const int kmax = max(max(padded(P.H, F), padded(P.nq * P.d, F)), padded(P.ncols, F));
  const int attn = attn_lds_floats(P.d, P.nchunk);
  uint16_t* xs = reinterpret_cast<uint16_t*>(lds);  // fp16 GEMV input (kmax halfs)
  float* slots = lds + max(kmax / 2, attn);
  float* red = slots + MAX_SLOTS;
  run_phases<PB, PE, PB, F>(P, lds, xs, slots, red);
  if constexpr (PE > PB) grid_exit(P.sync);
}

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

  // router logits (xs keeps w for the gate/up phase)
  gemv_phase<1, FMT_F16>(
      RowsOne{make_mat(P.wr, P.ld_r, P.E, nullptr, 0)}, P.E, P.H, xs, slots, nullptr,
      [&]() { stage_rmsnorm_h(P.h, P.g_ffn, P.H, padded(P.H, FMT_F16), P.eps, xs, red); },
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

typedef void (*DecodeKernel)(Params);

// Instantiations: the whole step, each sub-layer, and each phase alone.
template <int F>
__host__ inline DecodeKernel decode_kernel_fmt(int pb, int pe) {
  if (pb == PH_QKV && pe == PH_DOWN) return decode_kernel<PH_QKV, PH_DOWN, F>;
  if (pb == PH_QKV && pe == PH_O) return decode_kernel<PH_QKV, PH_O, F>;
  if (pb == PH_GATEUP && pe == PH_DOWN) return decode_kernel<PH_GATEUP, PH_DOWN, F>;
  if (pb == pe) {
    switch (pb) {
      case PH_QKV: return decode_kernel<PH_QKV, PH_QKV, F>;
      case PH_ATTN: return decode_kernel<PH_ATTN, PH_ATTN, F>;
      case PH_O: return decode_kernel<PH_O, PH_O, F>;
      case PH_GATEUP: return decode_kernel<PH_GATEUP, PH_GATEUP, F>;
      case PH_DOWN: return decode_kernel<PH_DOWN, PH_DOWN, F>;
    }
  }
  return nullptr;
}

__host__ inline DecodeKernel decode_kernel_for(int pb, int pe, int fmt) {
  switch (fmt) {
    case FMT_F16: return decode_kernel_fmt<FMT_F16>(pb, pe);
    case FMT_Q8: return decode_kernel_fmt<FMT_Q8>(pb, pe);
    case FMT_Q4: return decode_kernel_fmt<FMT_Q4>(pb, pe);
  }
  return nullptr;
}

// ---------------------------------------------------------------------------
// KV append: a pure copy of n_tok tokens into every KV head's slots
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256) kv_append_kernel(const uint16_t* __restrict__ k,
                                                        const uint16_t* __restrict__ v,
                                                        uint16_t* __restrict__ kc,
                                                        uint16_t* __restrict__ vc, int n_tok,
                                                        int nkv, int d, int cap, int pos) {
  const int per_tok = nkv * d / 8;
  const int64_t total = static_cast<int64_t>(n_tok) * per_tok;
  for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < total;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int tok = static_cast<int>(i / per_tok);
    const int rem = static_cast<int>(i - static_cast<int64_t>(tok) * per_tok);
    const int g = rem / (d / 8), c8 = rem - g * (d / 8);
    const int64_t src = static_cast<int64_t>(tok) * nkv * d + static_cast<int64_t>(g) * d + c8 * 8;
    const int64_t dst = (static_cast<int64_t>(g) * cap + pos + tok) * d + c8 * 8;
    *reinterpret_cast<u32x4*>(kc + dst) = *reinterpret_cast<const u32x4*>(k + src);
    *reinterpret_cast<u32x4*>(vc + dst) = *reinterpret_cast<const u32x4*>(v + src);
  }
}

}  // namespace dec

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
namespace {

struct DeviceInfo {
  int cus = 0;
  size_t max_lds = 0;
  bool lds_attr_set = false;
};

std::mutex g_dev_mu;
std::vector<DeviceInfo> g_dev;

vt_status device_info(DeviceInfo** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(VT_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  std::lock_guard<std::mutex> lk(g_dev_mu);
  if (static_cast<int>(g_dev.size()) <= dev) g_dev.resize(dev + 1);
  DeviceInfo& di = g_dev[dev];
  if (di.cus == 0) {
    int cus = 0, lds = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return fail(VT_ERR_HIP, "hipDeviceGetAttribute: %s", hipGetErrorString(e));
    e = hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
    if (e != hipSuccess) return fail(VT_ERR_HIP, "hipDeviceGetAttribute: %s", hipGetErrorString(e));
    di.cus = cus;
    di.max_lds = static_cast<size_t>(lds);
  }
  if (!di.lds_attr_set) {
    // Allow dynamic LDS up to the device limit; a refusal surfaces as a
    // launch error for the shapes that would need it.
    const int ranges[][2] = {{0, 4}, {0, 2}, {3, 4}, {0, 0}, {1, 1}, {2, 2}, {3, 3}, {4, 4}};
    for (int fmt : {dec::FMT_F16, dec::FMT_Q8, dec::FMT_Q4})
      for (const auto& r : ranges)
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(dec::decode_kernel_for(r[0], r[1], fmt)),
                                  hipFuncAttributeMaxDynamicSharedMemorySize,
                                  static_cast<int>(di.max_lds));
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(dec::moe_kernel),
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(di.max_lds));
    (void)hipGetLastError();
    di.lds_attr_set = true;
  }
  *out = &di;
  return VT_OK;
}

inline int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

}  // namespace

// Workspace layout of the decode path (bytes, each region 256-aligned).
struct DecodeWs {
  size_t sync, qkv, part, o, m, hbuf, total;
};

// Chunking of the attention phase: the chunk length is a whole number of
// passes (at most MAXPASS) chosen so that the (query head, chunk) items fill
// the grid about once.
static void attn_chunking(int d, int nq, int L, int grid, int* cl, int* nchunk) {
  const int ppp = dec::attn_ppp(d);
  const int target = std::max(1, grid / std::max(1, nq));
  int passes = (L + ppp * target - 1) / (ppp * target);
  passes = std::min(dec::MAXPASS, std::max(1, passes));
  *cl = passes * ppp;
  *nchunk = (L + *cl - 1) / *cl;
}

static DecodeWs decode_ws_layout(const vt_shard_spec& s, int32_t max_ctx) {
  const vt_shard_info& in = s.info;
  const int d = s.dims.head_dim;
  const int64_t nchunk = (max_ctx + dec::attn_ppp(d) - 1) / dec::attn_ppp(d);
  DecodeWs w{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off += static_cast<size_t>(round_up(static_cast<int64_t>(bytes), 256));
    return at;
  };
  w.sync = take(sizeof(unsigned) * (dec::SW_GROUP + (in.n_q_heads + 1) * dec::SW_GROUP_STRIDE));
  w.qkv = take(sizeof(float) * (in.n_q_heads + 2 * in.n_kv_heads) * d);
  w.part = take(sizeof(float) * in.n_q_heads * nchunk * (d + dec::REC));
  w.o = take(sizeof(float) * in.n_q_heads * d);
  w.m = take(sizeof(float) * (in.n_cols + 8));
  w.hbuf = take(sizeof(float) * s.dims.hidden);
  w.total = off;
  return w;
}

size_t decode_workspace_bytes(const vt_shard_spec& s, int32_t max_ctx) {
  return decode_ws_layout(s, max_ctx).total;
}

// The synchronisation words sit at the start of the workspace; every other
// entry point keeps its buffers past them.
size_t workspace_sync_bytes(const vt_shard_spec& s) { return decode_ws_layout(s, 1).qkv; }

vt_status check_weights(const vt_shard_spec& s, const vt_layer_weights* w, bool attn, bool ffn) {
  if (!w) return fail(VT_ERR_ARG, "null weights");
  const int H = s.dims.hidden, d = s.dims.head_dim;
  const vt_shard_info& in = s.info;
  auto mat = [&](const void* p, int64_t ld, int64_t rowlen, int64_t rows, const char* name) -> vt_status {
    if (!p) return fail(VT_ERR_ARG, "weight %s is NULL", name);
    if (rows * ld * 2 >= kMaxBufferBytes)
      return fail(VT_ERR_UNSUPPORTED, "weight %s spans %lld bytes; the kernels address < 2 GiB", name,
                  static_cast<long long>(rows * ld * 2));
    if (!aligned16(p)) return fail(VT_ERR_ALIGN, "weight %s is not 16-byte aligned", name);
    if (ld < rowlen) return fail(VT_ERR_ARG, "ld of %s (%lld) < row length %lld", name,
                                 static_cast<long long>(ld), static_cast<long long>(rowlen));
    if (ld % 8) return fail(VT_ERR_ALIGN, "ld of %s (%lld) is not a multiple of 8", name,
                            static_cast<long long>(ld));
    return VT_OK;
  };
  auto gain = [&](const void* p, const char* name) -> vt_status {
    if (!p) return fail(VT_ERR_ARG, "gain %s is NULL", name);
    if (!aligned16(p)) return fail(VT_ERR_ALIGN, "gain %s is not 16-byte aligned", name);
    return VT_OK;
  };
  vt_status st;
  if (attn) {
    if ((st = gain(w->g_attn, "g_attn")) != VT_OK) return st;
    if (in.n_q_heads > 0) {
      const int64_t qd = static_cast<int64_t>(in.n_q_heads) * d;
      const int64_t kd = static_cast<int64_t>(in.n_kv_heads) * d;
      if ((st = mat(w->wq, w->ld_q, H, qd, "wq")) != VT_OK) return st;
      if ((st = mat(w->wk, w->ld_k, H, kd, "wk")) != VT_OK) return st;
      if ((st = mat(w->wv, w->ld_v, H, kd, "wv")) != VT_OK) return st;
      if ((st = mat(w->wo, w->ld_o, qd, H, "wo")) != VT_OK) return st;
    }
  }
  if (ffn) {
    if ((st = gain(w->g_ffn, "g_ffn")) != VT_OK) return st;
    if (in.n_cols > 0) {
      if ((st = mat(w->wg, w->ld_g, H, in.n_cols, "wg")) != VT_OK) return st;
      if ((st = mat(w->wu, w->ld_u, H, in.n_cols, "wu")) != VT_OK) return st;
      if ((st = mat(w->wd, w->ld_d, in.n_cols, H, "wd")) != VT_OK) return st;
    }
  }
  return VT_OK;
}

// Block-quantised weights: per matrix the codes (16-byte aligned rows of at
// least the row's code bytes) and the scales (2-byte aligned, at least one
// per block), each within the 2 GiB a buffer resource addresses.
static vt_status check_qweights(const vt_shard_spec& s, const vt_layer_qweights* w, bool attn, bool ffn) {
  if (!w) return fail(VT_ERR_ARG, "null weights");
  if (w->prec != VT_W_INT8 && w->prec != VT_W_INT4)
    return fail(VT_ERR_ARG, "weight precision %d is neither VT_W_INT8 nor VT_W_INT4", w->prec);
  const int H = s.dims.hidden, d = s.dims.head_dim;
  const vt_shard_info& in = s.info;
  // a row's block scales are staged in LDS, at most 512 of them
  const int64_t kmax = std::max({static_cast<int64_t>(H), static_cast<int64_t>(in.n_q_heads) * d,
                                 static_cast<int64_t>(in.n_cols)});
  if (kmax > 16384)
    return fail(VT_ERR_UNSUPPORTED, "quantised rows of %lld columns; at most 16384",
                static_cast<long long>(kmax));
  auto mat = [&](const vt_qmat& m, int64_t rowlen, int64_t rows, const char* name) -> vt_status {
    const int64_t nb = (rowlen + 31) / 32;
    const int64_t need = nb * (w->prec == VT_W_INT8 ? 32 : 16);
    if (!m.codes || !m.scales) return fail(VT_ERR_ARG, "codes or scales of %s are NULL", name);
    if (!aligned16(m.codes)) return fail(VT_ERR_ALIGN, "codes of %s are not 16-byte aligned", name);
    if (reinterpret_cast<uintptr_t>(m.scales) % 2)
      return fail(VT_ERR_ALIGN, "scales of %s are not 2-byte aligned", name);
    if (m.ld_codes < need || m.ld_codes % 16)
      return fail(VT_ERR_ARG, "ld_codes of %s (%lld) must be a multiple of 16 and >= %lld", name,
                  static_cast<long long>(m.ld_codes), static_cast<long long>(need));
    if (m.ld_scales < nb)
      return fail(VT_ERR_ARG, "ld_scales of %s (%lld) < %lld blocks", name,
                  static_cast<long long>(m.ld_scales), static_cast<long long>(nb));
    if (rows * m.ld_codes >= kMaxBufferBytes || rows * m.ld_scales * 2 >= kMaxBufferBytes)
      return fail(VT_ERR_UNSUPPORTED, "weight %s spans 2 GiB or more; the kernels address < 2 GiB", name);
    return VT_OK;
  };
  auto gain = [&](const void* p, const char* name) -> vt_status {
    if (!p) return fail(VT_ERR_ARG, "gain %s is NULL", name);
    if (!aligned16(p)) return fail(VT_ERR_ALIGN, "gain %s is not 16-byte aligned", name);
    return VT_OK;
  };
  vt_status st;
  if (attn) {
    if ((st = gain(w->g_attn, "g_attn")) != VT_OK) return st;
    if (in.n_q_heads > 0) {
      const int64_t qd = static_cast<int64_t>(in.n_q_heads) * d;
      const int64_t kd = static_cast<int64_t>(in.n_kv_heads) * d;
      if ((st = mat(w->wq, H, qd, "wq")) != VT_OK) return st;
      if ((st = mat(w->wk, H, kd, "wk")) != VT_OK) return st;
      if ((st = mat(w->wv, H, kd, "wv")) != VT_OK) return st;
      if ((st = mat(w->wo, qd, H, "wo")) != VT_OK) return st;
    }
  }
  if (ffn) {
    if ((st = gain(w->g_ffn, "g_ffn")) != VT_OK) return st;
    if (in.n_cols > 0) {
      if ((st = mat(w->wg, H, in.n_cols, "wg")) != VT_OK) return st;
      if ((st = mat(w->wu, H, in.n_cols, "wu")) != VT_OK) return st;
      if ((st = mat(w->wd, in.n_cols, H, "wd")) != VT_OK) return st;
    }
  }
  return VT_OK;
}

vt_status check_kv(const vt_shard_spec& s, const vt_kv_view* kv, int32_t pos, int32_t n_tok) {
  if (!kv) return fail(VT_ERR_ARG, "null KV view");
  if (kv->n_kv_heads != s.info.n_kv_heads || kv->head_dim != s.dims.head_dim)
    return fail(VT_ERR_ARG, "KV view has %d heads x %d dims, shard needs %d x %d", kv->n_kv_heads,
                kv->head_dim, s.info.n_kv_heads, s.dims.head_dim);
  if (kv->capacity < 1 || kv->len < 0 || kv->len > kv->capacity)
    return fail(VT_ERR_ARG, "KV view capacity %d / len %d invalid", kv->capacity, kv->len);
  if (static_cast<int64_t>(kv->n_kv_heads) * kv->capacity * kv->head_dim * 2 >= kMaxBufferBytes)
    return fail(VT_ERR_UNSUPPORTED, "KV cache of %d heads x %d positions exceeds 2 GiB per tensor",
                kv->n_kv_heads, kv->capacity);
  if (s.info.n_kv_heads > 0) {
    if (!kv->k || !kv->v) return fail(VT_ERR_ARG, "KV buffers are NULL");
    if (!aligned16(kv->k) || !aligned16(kv->v)) return fail(VT_ERR_ALIGN, "KV buffers not 16-byte aligned");
  }
  if (pos != kv->len) return fail(VT_ERR_POS, "pos %d != KV length %d", pos, kv->len);
  if (n_tok < 0 || static_cast<int64_t>(pos) + n_tok > kv->capacity)
    return fail(VT_ERR_KV_FULL, "appending %d tokens at %d passes capacity %d", n_tok, pos,
                kv->capacity);
  return VT_OK;
}

}  // namespace vt

using namespace vt;

static vt_status check_io_vec(const void* p, const char* name, bool required) {
  if (!p) return required ? fail(VT_ERR_ARG, "%s is NULL", name) : VT_OK;
  if (!aligned16(p)) return fail(VT_ERR_ALIGN, "%s is not 16-byte aligned", name);
  return VT_OK;
}

extern "C" vt_status vt_kv_append(vt_kv_view* kv, const void* k, const void* v, int32_t n_tok,
                                  int32_t pos, void* stream) {
  clear_error();
  if (!kv) return fail(VT_ERR_ARG, "null KV view");
  if (n_tok < 0) return fail(VT_ERR_ARG, "n_tok %d < 0", n_tok);
  if (kv->head_dim != 64 && kv->head_dim != 128)
    return fail(VT_ERR_UNSUPPORTED, "head_dim %d", kv->head_dim);
  if (kv->n_kv_heads < 0 || kv->capacity < 1 || kv->len < 0 || kv->len > kv->capacity)
    return fail(VT_ERR_ARG, "KV view fields invalid");
  if (pos != kv->len) return fail(VT_ERR_POS, "pos %d != KV length %d", pos, kv->len);
  if (static_cast<int64_t>(pos) + n_tok > kv->capacity)
    return fail(VT_ERR_KV_FULL, "appending %d tokens at %d passes capacity %d", n_tok, pos,
                kv->capacity);
  if (n_tok == 0 || kv->n_kv_heads == 0) {
    kv->len = pos + n_tok;
    return VT_OK;
  }
  if (!k || !v || !kv->k || !kv->v) return fail(VT_ERR_ARG, "null buffer");
  if (!aligned16(k) || !aligned16(v) || !aligned16(kv->k) || !aligned16(kv->v))
    return fail(VT_ERR_ALIGN, "buffers must be 16-byte aligned");
  const int64_t chunks = static_cast<int64_t>(n_tok) * kv->n_kv_heads * kv->head_dim / 8;
  const int blocks = static_cast<int>(std::min<int64_t>((chunks + 255) / 256, 4096));
  hipLaunchKernelGGL(dec::kv_append_kernel, dim3(blocks), dim3(256), 0,
                     static_cast<hipStream_t>(stream), static_cast<const uint16_t*>(k),
                     static_cast<const uint16_t*>(v), static_cast<uint16_t*>(kv->k),
                     static_cast<uint16_t*>(kv->v), n_tok, kv->n_kv_heads, kv->head_dim,
                     kv->capacity, pos);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(VT_ERR_HIP, "kv_append launch: %s", hipGetErrorString(e));
  kv->len = pos + n_tok;
  return VT_OK;
}

// The weights of a decode call in a format-neutral view: per matrix (q, k,
// v, o, gate, up, down) the values or codes and their row stride in bytes,
// and for the quantised formats the block scales and their stride in bytes.
struct WeightView {
  int fmt;
  const void *g_attn, *g_ffn;
  const void* w[7];
  int64_t ld[7];
  const void* sc[7];
  int64_t lds[7];
};

static vt_status decode_impl(const vt_shard_spec* spec, const WeightView& W, vt_kv_view* kv,
                             const vt_layer_io* io, int32_t pos, uint32_t phases, void* ws,
                             size_t ws_bytes, void* stream);

static vt_status check_phases(const vt_shard_spec* spec, const vt_layer_io* io, uint32_t phases) {
  if (!spec || !io) return fail(VT_ERR_ARG, "null spec or io");
  if (phases & ~(VT_ATTN | VT_FFN | VT_STAGED)) return fail(VT_ERR_ARG, "unknown phase bits 0x%x", phases);
  if (!(phases & (VT_ATTN | VT_FFN))) return fail(VT_ERR_ARG, "no phase selected");
  return VT_OK;
}

extern "C" vt_status vt_layer_decode(const vt_shard_spec* spec, const vt_layer_weights* w,
                                     vt_kv_view* kv, const vt_layer_io* io, int32_t pos,
                                     uint32_t phases, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  vt_status st = check_phases(spec, io, phases);
  if (st != VT_OK) return st;
  if ((st = check_weights(*spec, w, phases & VT_ATTN, phases & VT_FFN)) != VT_OK) return st;
  WeightView W{};
  W.fmt = dec::FMT_F16;
  W.g_attn = w->g_attn;
  W.g_ffn = w->g_ffn;
  const void* ptrs[7] = {w->wq, w->wk, w->wv, w->wo, w->wg, w->wu, w->wd};
  const int64_t lds[7] = {w->ld_q, w->ld_k, w->ld_v, w->ld_o, w->ld_g, w->ld_u, w->ld_d};
  for (int i = 0; i < 7; ++i) {
    W.w[i] = ptrs[i];
    W.ld[i] = lds[i] * 2;
  }
  return decode_impl(spec, W, kv, io, pos, phases, ws, ws_bytes, stream);
}

extern "C" vt_status vt_layer_decode_q(const vt_shard_spec* spec, const vt_layer_qweights* w,
                                       vt_kv_view* kv, const vt_layer_io* io, int32_t pos,
                                       uint32_t phases, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  vt_status st = check_phases(spec, io, phases);
  if (st != VT_OK) return st;
  if ((st = check_qweights(*spec, w, phases & VT_ATTN, phases & VT_FFN)) != VT_OK) return st;
  WeightView W{};
  W.fmt = w->prec == VT_W_INT8 ? dec::FMT_Q8 : dec::FMT_Q4;
  W.g_attn = w->g_attn;
  W.g_ffn = w->g_ffn;
  const vt_qmat* m[7] = {&w->wq, &w->wk, &w->wv, &w->wo, &w->wg, &w->wu, &w->wd};
  for (int i = 0; i < 7; ++i) {
    W.w[i] = m[i]->codes;
    W.ld[i] = m[i]->ld_codes;
    W.sc[i] = m[i]->scales;
    W.lds[i] = m[i]->ld_scales * 2;
  }
  return decode_impl(spec, W, kv, io, pos, phases, ws, ws_bytes, stream);
}

static vt_status decode_impl(const vt_shard_spec* spec, const WeightView& W, vt_kv_view* kv,
                             const vt_layer_io* io, int32_t pos, uint32_t phases, void* ws,
                             size_t ws_bytes, void* stream) {
  const bool attn = phases & VT_ATTN, ffn = phases & VT_FFN, staged = phases & VT_STAGED;
  const vt_layer_dims& D = spec->dims;
  const vt_shard_info& in = spec->info;
  vt_status st = VT_OK;
  if (attn) {
    if ((st = check_kv(*spec, kv, pos, 1)) != VT_OK) return st;
    if ((st = check_io_vec(io->x, "x", true)) != VT_OK) return st;
    if ((st = check_io_vec(io->peer_attn, "peer_attn", false)) != VT_OK) return st;
    if ((st = check_io_vec(io->attn_partial, "attn_partial", true)) != VT_OK) return st;
  }
  if ((st = check_io_vec(io->h, "h", true)) != VT_OK) return st;
  if (ffn) {
    if ((st = check_io_vec(io->peer_ffn, "peer_ffn", false)) != VT_OK) return st;
    if ((st = check_io_vec(io->ffn_partial, "ffn_partial", true)) != VT_OK) return st;
    if ((st = check_io_vec(io->y, "y", false)) != VT_OK) return st;
  }
  const int ctx = attn ? pos + 1 : 1;
  // a sliding window attends to the last D.window positions only
  const int p_first = (attn && D.window > 0) ? std::max(0, pos + 1 - D.window) : 0;
  const DecodeWs L = decode_ws_layout(*spec, ctx);
  if (!ws || ws_bytes < L.total)
    return fail(VT_ERR_WORKSPACE, "workspace %zu bytes, need %zu", ws_bytes, L.total);
  if (!aligned16(ws)) return fail(VT_ERR_ALIGN, "workspace not 16-byte aligned");

  DeviceInfo* di = nullptr;
  if ((st = device_info(&di)) != VT_OK) return st;

  dec::Params P{};
  P.H = D.hidden;
  P.d = D.head_dim;
  P.nq = in.n_q_heads;
  P.nkv = in.n_kv_heads;
  P.G = D.n_heads / D.n_kv_heads;
  P.ncols = in.n_cols;
  P.pos = pos;
  P.p_first = p_first;
  P.cap = kv ? kv->capacity : 0;
  attn_chunking(D.head_dim, in.n_q_heads, ctx - p_first, di->cus, &P.cl, &P.nchunk);
  P.eps = D.rms_eps;
  P.rope_base = D.rope_base;
  P.g_attn = static_cast<const uint16_t*>(W.g_attn);
  P.g_ffn = static_cast<const uint16_t*>(W.g_ffn);
  const uint8_t** wp[7] = {&P.wq, &P.wk, &P.wv, &P.wo, &P.wg, &P.wu, &P.wd};
  int64_t* ldp[7] = {&P.ld_q, &P.ld_k, &P.ld_v, &P.ld_o, &P.ld_g, &P.ld_u, &P.ld_d};
  const uint16_t** sp[7] = {&P.sq, &P.sk, &P.sv, &P.so, &P.sg, &P.su, &P.sd};
  int64_t* lsp[7] = {&P.lds_q, &P.lds_k, &P.lds_v, &P.lds_o, &P.lds_g, &P.lds_u, &P.lds_d};
  for (int i = 0; i < 7; ++i) {
    *wp[i] = static_cast<const uint8_t*>(W.w[i]);
    *ldp[i] = W.ld[i];
    *sp[i] = static_cast<const uint16_t*>(W.sc[i]);
    *lsp[i] = W.lds[i];
  }
  P.kc = kv ? static_cast<uint16_t*>(kv->k) : nullptr;
  P.vc = kv ? static_cast<uint16_t*>(kv->v) : nullptr;
  P.kv_bytes = kv ? static_cast<uint32_t>(static_cast<int64_t>(kv->n_kv_heads) * kv->capacity *
                                          kv->head_dim * 2)
                  : 0u;
  P.x = static_cast<const uint16_t*>(io->x);
  P.peer_a = static_cast<const uint16_t*>(io->peer_attn);
  P.peer_f = static_cast<const uint16_t*>(io->peer_ffn);
  P.p_attn = static_cast<uint16_t*>(io->attn_partial);
  P.h = static_cast<uint16_t*>(io->h);
  P.p_ffn = static_cast<uint16_t*>(io->ffn_partial);
  P.y = static_cast<uint16_t*>(io->y);
  char* base = static_cast<char*>(ws);
  P.sync = reinterpret_cast<unsigned*>(base + L.sync);
  P.qkv = reinterpret_cast<float*>(base + L.qkv);
  P.part = reinterpret_cast<float*>(base + L.part);
  P.o = reinterpret_cast<float*>(base + L.o);
  P.m = reinterpret_cast<float*>(base + L.m);
  P.hbuf = reinterpret_cast<float*>(base + L.hbuf);
  P.h_from_ws = attn ? 1 : 0;

  const int kmax = std::max({dec::padded(P.H, W.fmt), dec::padded(P.nq * P.d, W.fmt),
                             dec::padded(P.ncols, W.fmt)});
  const int attn_f = dec::attn_lds_floats(P.d, P.nchunk);
  const size_t lds = sizeof(float) * (std::max(kmax / 2, attn_f) + dec::MAX_SLOTS + 16) +
                     (W.fmt == dec::FMT_F16 ? 0 : sizeof(uint16_t) * dec::SC_LDS_HALFS);
  if (lds > di->max_lds)
    return fail(VT_ERR_UNSUPPORTED, "shape needs %zu bytes of LDS, device has %zu", lds, di->max_lds);

  const int pb = attn ? dec::PH_QKV : dec::PH_GATEUP;
  const int pe = ffn ? dec::PH_DOWN : dec::PH_O;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipSuccess;
  if (staged) {
    for (int ph = pb; ph <= pe && e == hipSuccess; ++ph) {
      P.phase_begin = P.phase_end = ph;
      hipLaunchKernelGGL(dec::decode_kernel_for(ph, ph, W.fmt), dim3(di->cus), dim3(dec::NT), lds, s, P);
      e = hipGetLastError();
    }
  } else {
    // The grid barrier needs every workgroup resident at once: one per CU,
    // and the occupancy query confirms a CU holds at least one. A plain
    // launch is used (the cooperative launch API adds ~20 us per launch);
    // the barrier's bounded wait reports rather than hangs if another
    // kernel were to hold CUs.
    const dec::DecodeKernel kern = dec::decode_kernel_for(pb, pe, W.fmt);
    int per_cu = 0;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, dec::NT, lds);
    if (e != hipSuccess) return fail(VT_ERR_HIP, "occupancy query: %s", hipGetErrorString(e));
    if (per_cu < 1)
      return fail(VT_ERR_UNSUPPORTED, "decode kernel does not fit on a CU with %zu bytes of LDS", lds);
    P.phase_begin = pb;
    P.phase_end = pe;
    hipLaunchKernelGGL(kern, dim3(di->cus), dim3(dec::NT), lds, s, P);
    e = hipGetLastError();
  }
  if (e != hipSuccess) return fail(VT_ERR_HIP, "decode launch: %s", hipGetErrorString(e));
  if (attn) kv->len = pos + 1;
  return VT_OK;
}

extern "C" vt_status vt_workspace_size(const vt_shard_spec* spec, int32_t max_tokens,
                                       int32_t max_ctx, size_t* bytes) {
  clear_error();
  if (!spec || !bytes) return fail(VT_ERR_ARG, "null argument");
  if (max_tokens < 1 || max_ctx < 1) return fail(VT_ERR_ARG, "max_tokens and max_ctx must be >= 1");
  *bytes = std::max(decode_workspace_bytes(*spec, max_ctx),
                    prefill_workspace_bytes(*spec, max_tokens, max_ctx));
  return VT_OK;
}

// ---------------------------------------------------------------------------
// MoE FFN of a shard
// ---------------------------------------------------------------------------
namespace {

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
  DeviceInfo* di = nullptr;
  if ((st = device_info(&di)) != VT_OK) return st;

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
