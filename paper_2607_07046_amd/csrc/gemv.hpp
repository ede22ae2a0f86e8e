// Device building blocks shared by the decode and MoE kernels: the
// persistent grid's barrier, the weight-streaming GEMV phase (fp16 and
// block-quantised INT8 / INT4 rows) and the staging of a phase's input
// vector into LDS. Everything here runs inside one persistent launch of one
// 512-thread workgroup per CU.
#pragma once

#include <hip/hip_runtime.h>

#include "device.hpp"

namespace vt {
namespace dec {

constexpr int NT = 512;          // threads per workgroup (8 waves)
constexpr int NW = NT / kWave;   // waves per workgroup
constexpr int PF = 16;           // pieces in flight per wave
constexpr int PRE = 16;          // of which issued before the phase's barrier wait
constexpr int MAX_SLOTS = 4096;  // pieces per workgroup round (one float each)
constexpr unsigned kSpinLimit = 1u << 20;  // about a second of polling

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

// One GEMV phase over ``units`` output units of U virtual rows of K columns.
// A row is split into segments (512 fp16, 1024 INT8 or 2048 INT4 columns);
// a piece is one segment of one row (64 lanes x 16 B). The units are split
// evenly over the workgroups; a workgroup's rows (in rounds of at most
// MAX_SLOTS pieces) form one contiguous run of pieces that its eight waves
// split into contiguous sub-runs. ``pre`` runs first (all threads; loads
// issued there leave ahead of every weight piece), each wave issues its
// first PRE pieces, then ``stage`` runs (all threads: it waits at the grid barrier in front of
// the phase, if any, writes the input as fp16 to xs16[0, nseg * SEGC), zero
// past K, and ends with a workgroup barrier), then the wave streams the rest
// of its sub-run through a ring of PF loads, accumulating a row's segments
// in each lane and reducing across the wave at the row's end (or where its
// sub-run ends) into slots[piece]. ``epi(unit, sums)`` gets each unit's U
// row sums, added in piece order (a fixed order: bitwise reproducible).
// With U == 32 (units of 32 rows) the epilogue is ``epi(unit, j, sum of row
// j)`` on lane j of a half-wave instead.
template <int U, int F, int SCW, class Rows, class Pre, class Stage, class Epi>
__device__ __forceinline__ void gemv_impl(const Rows& rows, int units, int K, const uint16_t* xs16,
                                          float* slots, uint16_t* scl, Pre pre, Stage stage, Epi epi) {
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
    bool ok = (p < q1) && (sg != nseg - 1 || lane_in_tail);
    if constexpr (Rows::kSlotTail) ok = ok && sg * SEGC + lane * EPL < rows.col_limit(sg);
    const uint32_t oob = static_cast<uint32_t>(!ok) << 31;
    return __builtin_amdgcn_raw_buffer_load_b128(ra.rs, (base + lane16) | oob, 0, 0);
  };
  pre();
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
    if constexpr (U == 32) {
      // a half-wave per unit, lane j taking its row j (the loop bound is
      // uniform over each half-wave, so the epilogue may use its shuffles)
      for (int lu = threadIdx.x / 32; lu < ub - ua; lu += NT / 32) {
        const int j = threadIdx.x % 32;
        float a = 0.f;
        if (K > 0) {
          const float* sl = slots + (lu * U + j) * nseg;
          for (int s = 0; s < nseg; ++s) a += sl[s];
        }
        epi(ua + lu, j, a);
      }
    } else {
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
    }
    lds_barrier();  // slots, scales and xs free for reuse
    ua = ub;
  } while (ua < u1);
}

template <int U, int F, class Rows, class Pre, class Stage, class Epi>
__device__ __forceinline__ void gemv_phase(const Rows& rows, int units, int K, const uint16_t* xs16,
                                           float* slots, uint16_t* scl, Pre pre, Stage stage, Epi epi) {
  if constexpr (F == FMT_F16) {
    gemv_impl<U, F, 1>(rows, units, K, xs16, slots, scl, pre, stage, epi);
  } else {
    const int words = ((K + 31) / 32 + 2 * kWave - 1) / (2 * kWave);  // per lane and scale row
    if (words <= 1)
      gemv_impl<U, F, 1>(rows, units, K, xs16, slots, scl, pre, stage, epi);
    else if (words <= 2)
      gemv_impl<U, F, 2>(rows, units, K, xs16, slots, scl, pre, stage, epi);
    else
      gemv_impl<U, F, SC_ROW_WORDS>(rows, units, K, xs16, slots, scl, pre, stage, epi);
  }
}

template <int U, int F, class Rows, class Stage, class Epi>
__device__ __forceinline__ void gemv_phase(const Rows& rows, int units, int K, const uint16_t* xs16,
                                           float* slots, uint16_t* scl, Stage stage, Epi epi) {
  gemv_phase<U, F>(rows, units, K, xs16, slots, scl, []() {}, stage, epi);
}

// ---------------------------------------------------------------------------
// staging of a GEMV phase's input vector into LDS as fp16 (all threads; each
// ends with a workgroup barrier)
// ---------------------------------------------------------------------------
// xs[k] = fp16(v[k] * rstd * g[k]), rstd = 1 / sqrt(mean(v^2) + eps), for a
// caller-provided fp16 vector v (n a multiple of 8, n <= 8 * 4 * NT); zero
// for n <= k < npad.
template <int MAXC>
struct RmsInH {
  u32x4 xv[MAXC], gv[MAXC];
  // the loads (chunks past n read as zero)
  __device__ __forceinline__ void load(const uint16_t* v, const uint16_t* g, int n) {
    const rsrc_t rv = make_rsrc(v, static_cast<uint32_t>(n) * 2u);
    const rsrc_t rg = make_rsrc(g, static_cast<uint32_t>(n) * 2u);
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
      const uint32_t off = static_cast<uint32_t>(threadIdx.x + c * NT) * 16u;
      xv[c] = buf_load16(rv, off);
      gv[c] = buf_load16(rg, off);
    }
  }
  // the gains alone, and the vector alone (``shared``: written by other
  // workgroups of this launch, read through the agent-scope coherent path)
  __device__ __forceinline__ void load_g(const uint16_t* g, int n) {
    const rsrc_t rg = make_rsrc(g, static_cast<uint32_t>(n) * 2u);
#pragma unroll
    for (int c = 0; c < MAXC; ++c) gv[c] = buf_load16(rg, static_cast<uint32_t>(threadIdx.x + c * NT) * 16u);
  }
  __device__ __forceinline__ void load_x(const uint16_t* v, int n, bool shared) {
    const rsrc_t rv = make_rsrc(v, static_cast<uint32_t>(n) * 2u);
    if (shared) {
#pragma unroll
      for (int c = 0; c < MAXC; ++c)
        xv[c] = __builtin_amdgcn_raw_buffer_load_b128(rv, static_cast<uint32_t>(threadIdx.x + c * NT) * 16u, 0,
                                                      kCoherent);
    } else {
#pragma unroll
      for (int c = 0; c < MAXC; ++c) xv[c] = buf_load16(rv, static_cast<uint32_t>(threadIdx.x + c * NT) * 16u);
    }
  }
  // the norm and the fp16 writes to LDS
  __device__ __forceinline__ void finish(int n, int npad, float eps, uint16_t* xs, float* red) const {
    const int nch = n / 8;
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
};

template <int MAXC>
__device__ __forceinline__ void stage_rmsnorm_h_impl(const uint16_t* v, const uint16_t* g, int n, int npad,
                                                     float eps, uint16_t* xs, float* red) {
  RmsInH<MAXC> r;
  r.load(v, g, n);
  r.finish(n, npad, eps, xs, red);
}

// The same for an fp32 vector written by other workgroups of this launch
// (n a multiple of 8), each value first rounded to fp16: the value the
// caller's fp16 h would carry.
template <int MAXP>  // float pairs held per thread
__device__ __forceinline__ void stage_rmsnorm_f_impl(const float* v, const uint16_t* g, int n, int npad,
                                                     float eps, uint16_t* xs, float* red) {
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

// The staging loads of a vector written inside the launch go out in one
// batch with no per-lane guard (loads past the vector read zero), and each
// slot of the batch costs the CU's memory pipeline an instruction even when
// it reads nothing: the batch is sized for hidden sizes up to 8192 (a
// hidden size of 4096 uses half of it), the larger one taken only for
// longer vectors (8 instead of 16 pairs: 1.3 us per 7B step for h, 1.8 us
// for o and m).
__device__ __forceinline__ void stage_rmsnorm_h(const uint16_t* v, const uint16_t* g, int n, int npad,
                                                float eps, uint16_t* xs, float* red) {
  // (two chunks for hidden sizes up to 8192 measured 0.8 us slower per 7B
  // step: this staging waits behind the first weight pieces anyway)
  stage_rmsnorm_h_impl<4>(v, g, n, npad, eps, xs, red);
}

__device__ __forceinline__ void stage_rmsnorm_f(const float* v, const uint16_t* g, int n, int npad,
                                                float eps, uint16_t* xs, float* red) {
  if (n <= 2 * 8 * NT)
    stage_rmsnorm_f_impl<8>(v, g, n, npad, eps, xs, red);
  else
    stage_rmsnorm_f_impl<16>(v, g, n, npad, eps, xs, red);
}

// xs[k] = fp16(v[k]) for an fp32 vector written by other workgroups of this
// launch (its buffer holds an even number of floats); zero for n <= k < npad.
__device__ __forceinline__ void stage_copy_f(const float* v, int n, int npad, uint16_t* xs) {
  constexpr int MAXP = 8;  // pairs per thread and round trip (sized like the staging loads below)
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

}  // namespace dec
}  // namespace vt
