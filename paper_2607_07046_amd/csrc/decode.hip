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
// barrier; stream order then separates the phases. A launch may also run
// several consecutive layers of a stack (paper Sec. 2.1: identically shaped
// decoder layers are stacked; Sec. 3.2.1: the TP split repeats at every
// layer): layer l's output y is layer l+1's input x, handed over across a
// grid barrier like any other phase's input, so layer l+1's first QKV weight
// pieces are in flight before layer l has finished.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <mutex>
#include <vector>

#include "comm_block.hpp"
#include "device.hpp"
#include "gemv.hpp"
#include "internal.hpp"

namespace vt {
namespace dec {

constexpr int REC = 4;           // attention partial record = head_dim + REC floats
static_assert(SW_ERR * 4 == VT_WS_ERROR_WORD, "the error word's documented offset");

enum { PH_QKV = 0, PH_ATTN = 1, PH_O = 2, PH_GATEUP = 3, PH_DOWN = 4 };

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
  // Stacked layers: layer l's tensors sit l strides past layer 0's.
  int n_layers;        // layers run by one launch (1 unless a stack)
  int64_t lst_w[7];    // bytes between consecutive layers' q, k, v, o, gate, up, down values / codes
  int64_t lst_s[7];    // the same for their block scales
  int64_t lst_kv;      // elements between consecutive layers' K (and V) caches
  // Quantised emission of the partial sums (the COMM instantiation): plan
  // (precision and byte offset per block of 32) and message of each partial;
  // a NULL message is not emitted.
  const uint8_t *eprec_a, *eprec_f;
  const int32_t *eoff_a, *eoff_f;
  uint8_t *emsg_a, *emsg_f;
  uint32_t emsg_a_bytes, emsg_f_bytes;
};

// ---------------------------------------------------------------------------
// phase 1: attention
//
// Work item = (query head j, chunk of CL consecutive cached positions). A
// thread holds 8 of the d dimensions of one position per pass (d/8 threads
// per position, PPP positions per pass, CL = passes * PPP). The chunks
// cover the cached positions p_first..pos-1; the last chunk also takes the
// new token (its score in one extra slot), so a context of k * CL + 1
// positions needs k chunks, not k + 1. The chunk's keys and values do not
// depend on phase 0, so they are loaded into registers before the grid
// barrier. Items of the G query heads that share a KV head and a
// chunk are placed on workgroups with equal index mod 8, i.e. on one XCD, so
// the group reads each K/V tile from HBM once and from that XCD's L2 after.
// Each item writes (unnormalised sum of p*V, running max m, sum l); the last
// item of head j to finish merges the head's chunks by log-sum-exp.
// ---------------------------------------------------------------------------
constexpr int MAXPASS = 8;
// Chunks a merging thread loads per round trip (its group's chunks grp,
// grp + ngrp, ...): every slot issues its loads, and one past the last chunk
// still costs an instruction slot, so the batch is sized for the usual
// 17-26 chunks over 4 groups (16 measured 1.2 us slower per 7B step).
constexpr int MERGE_BATCH = 8;

__host__ __device__ __forceinline__ int attn_ppp(int d) { return NT / (d / 8); }

__host__ __device__ __forceinline__ int attn_lds_floats(int d, int nchunk) {
  const int ppp = attn_ppp(d);
  return d + MAXPASS * ppp + 4 + ppp * d + 2 * d + 2 * nchunk + 4;
}

template <class PT>
__device__ __forceinline__ void phase_attn(PT& P, int layer, float* lds, bool wait, unsigned nbar) {
  const int d = P.d, G = P.G, CL = P.cl;
  const int TPP = d / 8, PPP = NT / TPP, NPASS = CL / PPP;
  const int t = threadIdx.x, wave = t / kWave, lane = t % kWave;
  const int pl = t / TPP;             // position within a pass
  const int dc = (t % TPP) * 8;       // first of this thread's 8 dimensions
  const int RW = d + REC;             // floats per partial record
  const int units = P.nkv * P.nchunk; // (KV head, chunk) pairs
  const int ids = ((units + 7) / 8) * 8 * G;
  const float scale = 1.0f / sqrtf(static_cast<float>(d));
  // LDS (floats): qs[d] | S[MAXPASS*PPP + 4] | R[PPP*d] | kn[d] | vn[d] | W[2*nchunk] | flag
  // (S[CL]: the new token's score in the last chunk)
  float* qs = lds;
  float* S = qs + d;
  float* R = S + MAXPASS * PPP + 4;
  float* kn = R + PPP * d;
  float* vn = kn + d;
  float* W = vn + d;
  int* flag = reinterpret_cast<int*>(W + 2 * P.nchunk);
  uint16_t* const kcl = P.kc + layer * P.lst_kv;  // this layer's cache
  uint16_t* const vcl = P.vc + layer * P.lst_kv;
  const rsrc_t rk = make_rsrc(kcl, P.kv_bytes), rv = make_rsrc(vcl, P.kv_bytes);

  // rotation of pair t at the new position (independent of phase 0; the
  // same for every item)
  const int half = d / 2;
  float c0 = 1.f, s0 = 0.f;
  if (t < half) rope_angle(P.pos, t, d, P.rope_base, c0, s0);

  bool waited = false;
  for (int id = blockIdx.x;; id += gridDim.x) {
    // past the first item, leave as soon as none is left (the next item's
    // prologue would only delay this workgroup's arrival at the barrier,
    // and the last merges are on the step's critical path)
    if (waited && id >= ids) break;
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
    const bool has_new = c == P.nchunk - 1;  // the last chunk takes the new token
    if (has_new) {  // the new token's key (rotated) and value, rounded as stored
      const int64_t slot = (static_cast<int64_t>(g) * P.cap + P.pos) * d;
      const bool writer = jj == 0;  // one item per KV head appends to the cache
      if (t < half) {
        const float a = ka, b = kb;
        const uint16_t k0 = f2h(a * c0 - b * s0), k1 = f2h(a * s0 + b * c0);
        kn[2 * t] = h2f(k0);
        kn[2 * t + 1] = h2f(k1);
        if (writer) {
          kcl[slot + 2 * t] = k0;
          kcl[slot + 2 * t + 1] = k1;
        }
      } else if (t < half + d) {
        const int i = t - half;
        const uint16_t v0 = f2h(vv);
        vn[i] = h2f(v0);
        if (writer) vcl[slot + i] = v0;
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
        float sc = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) sc = fmaf(qs[dc + e], kf[e], sc);
        sc = group_sum(sc, TPP);
        if ((t % TPP) == 0) S[ps * PPP + pl] = p < P.pos ? sc : -INFINITY;  // cached positions only
      }
    }
    if (t < TPP) {  // the new token's score (its key as stored), in slot CL
      float sc = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) sc = fmaf(qs[dc + e], kn[dc + e], sc);
      sc = group_sum(sc, TPP);
      if (t == 0) S[CL] = has_new ? sc : -INFINITY;
    }
    __syncthreads();
    float* rec = P.part + (static_cast<int64_t>(j) * P.nchunk + c) * RW;
    if (wave == 0) {  // softmax statistics of the chunk
      float mx = -INFINITY;
      for (int q = lane; q <= CL; q += kWave) mx = fmaxf(mx, S[q]);
      mx = wave_max(mx);
      float l = 0.f;
      for (int q = lane; q <= CL; q += kWave) {
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
        const float e = S[ps * PPP + pl];
        float vf[8];
        unpack8(vr[ps], vf);
#pragma unroll
        for (int x = 0; x < 8; ++x) acc[x] = fmaf(e, vf[x], acc[x]);
      }
    }
    if (t < TPP && has_new) {  // the new token's value (position group 0)
      const float e = S[CL];
#pragma unroll
      for (int x = 0; x < 8; ++x) acc[x] = fmaf(e, vn[dc + x], acc[x]);
    }
    // two 16-byte stores per thread: eight scalar ones put a wave's 64
    // lanes on a few LDS banks (measured 1.0 us slower per step)
    *reinterpret_cast<f32x4*>(R + pl * d + dc) = f32x4{acc[0], acc[1], acc[2], acc[3]};
    *reinterpret_cast<f32x4*>(R + pl * d + dc + 4) = f32x4{acc[4], acc[5], acc[6], acc[7]};
    __syncthreads();
    // sum of R's PPP rows in two levels over all threads: group gi of the
    // NT / d groups adds rows gi, gi + NT / d, ... (PPP * d = 8 * NT, so 8
    // rows each, loads independent), then d threads add the group sums (a
    // one-thread-per-column loop over PPP rows was a chain of LDS round trips)
    {
      const int ng = NT / d, gi = t / d, dd = t % d;
      float a = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) a += R[(gi + ng * i) * d + dd];
      __syncthreads();
      R[gi * d + dd] = a;
      __syncthreads();
      if (t < d) {
        float s = 0.f;
        for (int q = 0; q < ng; ++q) s += R[q * d + t];
        st_shared(rec + t, s);
      }
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
      // (m, l, value[dd]) in batches of MERGE_BATCH (one round trip each) and keeps a
      // running (max, sum l, sum value) under the log-sum-exp rescaling; the
      // ngrp partial triples of each dd are then merged in a fixed order.
      const rsrc_t rj = make_rsrc(P.part + static_cast<int64_t>(j) * P.nchunk * RW,
                                  static_cast<uint32_t>(P.nchunk * RW) * 4u);
      const int ngrp = NT / d, grp = t / d, dd = t % d;
      float M = -INFINITY, Ls = 0.f, A = 0.f;
      for (int c0 = grp; grp < ngrp && c0 < P.nchunk; c0 += MERGE_BATCH * ngrp) {
        float mv[MERGE_BATCH], lv[MERGE_BATCH], ov[MERGE_BATCH];
#pragma unroll
        for (int u = 0; u < MERGE_BATCH; ++u) {  // unconditional; chunks past the last read zero
          const int cc = c0 + u * ngrp;
          const uint32_t rec = cc < P.nchunk ? static_cast<uint32_t>(cc * RW) * 4u : kOOB;
          buf_ld_shared2(rj, rec == kOOB ? kOOB : rec + d * 4u, mv[u], lv[u]);
          ov[u] = buf_ld_shared(rj, rec == kOOB ? kOOB : rec + dd * 4u);
        }
#pragma unroll
        for (int u = 0; u < MERGE_BATCH; ++u) {
          if (c0 + u * ngrp >= P.nchunk) {
            mv[u] = -INFINITY;
            lv[u] = 0.f;
            ov[u] = 0.f;
          }
        }
        float bm = M;
#pragma unroll
        for (int u = 0; u < MERGE_BATCH; ++u) bm = fmaxf(bm, mv[u]);
        const float r = M == -INFINITY ? 0.f : __expf(M - bm);
        Ls *= r;
        A *= r;
#pragma unroll
        for (int u = 0; u < MERGE_BATCH; ++u) {
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
// One phase of layer ``layer``; ``wait``: a grid barrier is in front of it,
// the ``nbar``-th of the launch. COMM: the O and down phases give each
// workgroup whole blocks of 32 output rows and emit the quantised partials.
template <int PH, int F, bool COMM, class PT>
__device__ __forceinline__ void run_phase(PT& P, int layer, float* lds, uint16_t* xs, float* slots,
                                          float* red, bool wait, unsigned nbar) {
  uint16_t* scl = reinterpret_cast<uint16_t*>(red + 16);  // block scales (quantised formats)
  // The fields that describe the weight matrices are read again in each
  // phase from the kernel-argument segment, through a pointer the compiler
  // cannot follow from one phase to the next (scalar loads): the buffer
  // descriptors built from them then live in scalar registers during their
  // own phase only. Kept live across the whole launch, they overflow the
  // scalar register file, and the spill reloads land in the weight-streaming
  // loops. The parameters are the kernel's only argument, so they start at
  // byte 0 of the segment.
  typedef const __attribute__((address_space(4))) uint32_t* KernargWords;
  KernargWords pk = (KernargWords)__builtin_amdgcn_kernarg_segment_ptr();
  asm volatile("" : "+s"(pk));
  static_assert(sizeof(Params) % 4 == 0, "Params is read as 32-bit words");
  uint32_t words[sizeof(Params) / 4];
#pragma unroll
  for (int i = 0; i < static_cast<int>(sizeof(Params) / 4); ++i) words[i] = pk[i];
  Params PW;
  __builtin_memcpy(&PW, words, sizeof(Params));
  // this layer's weight matrix i (values / codes and block scales)
  auto wmat = [&](int i, const uint8_t* w, int64_t ld, int64_t rows, const uint16_t* s, int64_t lds) {
    return make_mat(w + layer * PW.lst_w[i], ld, rows, s ? s + layer * (PW.lst_s[i] / 2) : s, lds);
  };
  const int64_t io = static_cast<int64_t>(layer) * P.H;  // this layer's vectors
  // the layer's input: the caller's x, or the previous layer's y written in
  // this launch (read through the coherent path)
  const bool x_shared = layer > 0;
  const uint16_t* x = x_shared ? P.y + io - P.H : P.x;
  if constexpr (PH == PH_QKV) {
    RowsQKV rows{wmat(0, PW.wq, PW.ld_q, PW.nq * PW.d, PW.sq, PW.lds_q),
                 wmat(1, PW.wk, PW.ld_k, PW.nkv * PW.d, PW.sk, PW.lds_k),
                 wmat(2, PW.wv, PW.ld_v, PW.nkv * PW.d, PW.sv, PW.lds_v), PW.nq * PW.d, PW.nkv * PW.d};
    // x and the gains depend on nothing in this launch: their loads go out
    // ahead of the first weight pieces instead of queueing behind them
    // (fp16 7B shard 47.6 -> 47.4 us, 70B 108.1 -> 106.4, INT4 40.9 -> 39.7;
    // INT8, whose scale rows also load up front, measured 43.7 -> 44.1 and
    // keeps them behind). A stacked layer's x is the previous layer's y:
    // only its gains can go early.
    constexpr bool kEarlyX = F != FMT_Q8;
    const uint16_t* g = P.g_attn + io;
    RmsInH<4> xin;
    gemv_phase<1, F>(
        rows, (P.nq + 2 * P.nkv) * P.d, P.H, xs, slots, scl,
        [&]() {
          if constexpr (kEarlyX) {
            if (x_shared)
              xin.load_g(g, P.H);
            else
              xin.load(x, g, P.H);
          }
        },
        [&]() {
          if (wait) grid_wait(P.sync, nbar);
          if constexpr (!kEarlyX) {
            if (x_shared) {
              xin.load_x(x, P.H, true);
              xin.load_g(g, P.H);
            } else {
              xin.load(x, g, P.H);
            }
          } else {
            if (x_shared) xin.load_x(x, P.H, true);
          }
          xin.finish(P.H, padded(P.H, F), P.eps, xs, red);
        },
        [&](int r, const float* v) { st_shared(P.qkv + r, v[0]); });
  } else if constexpr (PH == PH_ATTN) {
    phase_attn(P, layer, lds, wait, nbar);
  } else if constexpr (PH == PH_O) {
    RowsOne rows{wmat(3, PW.wo, PW.ld_o, PW.H, PW.so, PW.lds_o)};
    const int K = P.nq * P.d;
    uint16_t* const pa_out = P.p_attn + io;
    uint16_t* const h_out = P.h + io;
    const uint16_t* const peer = P.peer_a ? P.peer_a + io : nullptr;
    auto stage = [&]() {
      if (wait) grid_wait(P.sync, nbar);
      stage_copy_f(P.o, K, padded(K, F), xs);
    };
    auto epi = [&](int r, float pa) {
      pa_out[r] = f2h(pa);
      const float xr = h2f(x_shared ? ld_h16_shared(x + r) : x[r]);
      const float hv = xr + pa + (peer ? h2f(peer[r]) : 0.f);
      h_out[r] = f2h(hv);
      st_shared(P.hbuf + r, hv);
    };
    if constexpr (COMM) {
      // whole blocks of 32 rows per workgroup: the block's quantised message
      // (paper Sec. 4.3.2) leaves with the partial sums, lane j holding row j
      gemv_phase<32, F>(rows, P.H / 32, K, xs, slots, scl, stage, [&](int blk, int j, float v) {
        epi(blk * 32 + j, v);
        if (P.emsg_a)
          comm_encode_block_lanes(f2h(v), j, P.eprec_a[blk], P.eoff_a[blk],
                                  make_rsrc(P.emsg_a, P.emsg_a_bytes), P.emsg_a_bytes);
      });
    } else {
      gemv_phase<1, F>(rows, P.H, K, xs, slots, scl, stage, [&](int r, const float* v) { epi(r, v[0]); });
    }
  } else if constexpr (PH == PH_GATEUP) {
    RowsPair rows{wmat(4, PW.wg, PW.ld_g, PW.ncols, PW.sg, PW.lds_g),
                  wmat(5, PW.wu, PW.ld_u, PW.ncols, PW.su, PW.lds_u)};
    const uint16_t* const g = P.g_ffn + io;
    gemv_phase<2, F>(
        rows, P.ncols, P.H, xs, slots, scl,
        [&]() {
          if (wait) grid_wait(P.sync, nbar);
          if (P.h_from_ws)
            stage_rmsnorm_f(P.hbuf, g, P.H, padded(P.H, F), P.eps, xs, red);
          else
            stage_rmsnorm_h(P.h + io, g, P.H, padded(P.H, F), P.eps, xs, red);
        },
        [&](int j, const float* v) {
          const float gt = v[0], up = v[1];
          st_shared(P.m + j, gt / (1.0f + __expf(-gt)) * up);
        });
  } else {
    RowsOne rows{wmat(6, PW.wd, PW.ld_d, PW.H, PW.sd, PW.lds_d)};
    const int K = P.ncols;
    uint16_t* const pf_out = P.p_ffn + io;
    uint16_t* const y_out = P.y ? P.y + io : nullptr;
    const uint16_t* const peer = P.peer_f ? P.peer_f + io : nullptr;
    // a stacked layer's y is the next layer's x: written through the coherent path
    const bool y_shared = layer + 1 < P.n_layers;
    auto stage = [&]() {
      if (wait) grid_wait(P.sync, nbar);
      stage_copy_f(P.m, K, padded(K, F), xs);
    };
    auto epi = [&](int r, float pf) {
      pf_out[r] = f2h(pf);
      if (y_out) {
        const float hr = P.h_from_ws ? round_h(ld_shared(P.hbuf + r)) : h2f(P.h[io + r]);
        const uint16_t yv = f2h(hr + pf + (peer ? h2f(peer[r]) : 0.f));
        if (y_shared)
          st_h16_shared(y_out + r, yv);
        else
          y_out[r] = yv;
      }
    };
    if constexpr (COMM) {
      gemv_phase<32, F>(rows, P.H / 32, K, xs, slots, scl, stage, [&](int blk, int j, float v) {
        epi(blk * 32 + j, v);
        if (P.emsg_f)
          comm_encode_block_lanes(f2h(v), j, P.eprec_f[blk], P.eoff_f[blk],
                                  make_rsrc(P.emsg_f, P.emsg_f_bytes), P.emsg_f_bytes);
      });
    } else {
      gemv_phase<1, F>(rows, P.H, K, xs, slots, scl, stage, [&](int r, const float* v) { epi(r, v[0]); });
    }
  }
}

template <int PH, int PE, int PB, int F, bool COMM, class PT>
__device__ __forceinline__ void run_phases(PT& P, int layer, float* lds, uint16_t* xs, float* slots,
                                           float* red) {
  // barriers so far in this launch: (PE - PB + 1) per earlier layer
  const unsigned nbar = static_cast<unsigned>(layer * (PE - PB + 1) + PH - PB);
  run_phase<PH, F, COMM>(P, layer, lds, xs, slots, red, nbar > 0, nbar);
  if constexpr (PH < PE) {
    grid_arrive(P.sync);
    run_phases<PH + 1, PE, PB, F, COMM>(P, layer, lds, xs, slots, red);
  }
}

// Phases PB..PE of one decode step; with STACK, of each of P.n_layers
// stacked layers. PB < PE or STACK need every workgroup resident (one per
// CU): grid barriers separate the phases and the layers. Params must stay
// the only kernel argument (run_phase reads it from the start of the
// argument segment).
template <int PB, int PE, int F, bool STACK = false, bool COMM = false>
__global__ void __launch_bounds__(NT) decode_kernel(Params P) {
  extern __shared__ float lds[];
  // LDS: xs / attention scratch (aliased) | slots[MAX_SLOTS] | red[16] |
  // block scales (quantised formats)
  const int kmax = max(max(padded(P.H, F), padded(P.nq * P.d, F)), padded(P.ncols, F));
  const int attn = attn_lds_floats(P.d, P.nchunk);
  uint16_t* xs = reinterpret_cast<uint16_t*>(lds);  // fp16 GEMV input (kmax halfs)
  float* slots = lds + max(kmax / 2, attn);
  float* red = slots + MAX_SLOTS;
  if constexpr (STACK) {
    // Each layer reads the parameters through a pointer the compiler cannot
    // follow from one layer to the next: nothing computed from them is
    // hoisted out of the loop and kept live across every phase (which made
    // the register allocator spill vector registers to scratch).
    typedef const __attribute__((address_space(4))) Params KParams;
    for (int layer = 0; layer < P.n_layers; ++layer) {
      KParams* pp = (KParams*)__builtin_amdgcn_kernarg_segment_ptr();
      asm volatile("" : "+s"(pp));
      if (layer > 0) grid_arrive(pp->sync);
      run_phases<PB, PE, PB, F, COMM>(*pp, layer, lds, xs, slots, red);
    }
  } else {
    run_phases<PB, PE, PB, F, COMM>(P, 0, lds, xs, slots, red);
  }
  if constexpr (PE > PB || STACK) grid_exit(P.sync);
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

// The persistent kernel of a stack of fp16 layers (all phases, layer loop).
__host__ inline DecodeKernel decode_stack_kernel() { return decode_kernel<PH_QKV, PH_DOWN, FMT_F16, true>; }

// fp16 decode that also emits the quantised partial sums (persistent only).
__host__ inline DecodeKernel decode_comm_kernel(int pb, int pe) {
  if (pb == PH_QKV && pe == PH_DOWN) return decode_kernel<PH_QKV, PH_DOWN, FMT_F16, false, true>;
  if (pb == PH_QKV && pe == PH_O) return decode_kernel<PH_QKV, PH_O, FMT_F16, false, true>;
  if (pb == PH_GATEUP && pe == PH_DOWN) return decode_kernel<PH_GATEUP, PH_DOWN, FMT_F16, false, true>;
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

// Zero ``n`` 32-bit words (the synchronisation words of a workspace that
// may hold a previous call's contents).
__global__ void __launch_bounds__(256) zero_words(uint32_t* p, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0u;
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
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(dec::decode_stack_kernel()),
                              hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(di.max_lds));
    for (const auto& r : ranges)
      if (dec::decode_comm_kernel(r[0], r[1]))
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(dec::decode_comm_kernel(r[0], r[1])),
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

// Chunking of the attention phase over the L cached positions attended
// (the new token joins the last chunk): the chunk length is a whole number of
// passes (at most MAXPASS) chosen so that the (query head, chunk) items fill
// the grid about once.
static void attn_chunking(int d, int nq, int L, int grid, int* cl, int* nchunk) {
  const int ppp = dec::attn_ppp(d);
  const int target = std::max(1, grid / std::max(1, nq));
  int passes = (L + ppp * target - 1) / (ppp * target);
  passes = std::min(dec::MAXPASS, std::max(1, passes));
  *cl = passes * ppp;
  *nchunk = std::max(1, (L + *cl - 1) / *cl);
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

// A stack of layers in one launch: their count and the distances from one
// layer's tensors to the next's (bytes for the matrices, elements for the
// KV caches).
struct StackView {
  int n_layers = 1;
  int64_t lst_w[7] = {0, 0, 0, 0, 0, 0, 0};
  int64_t lst_kv = 0;
  bool clear_sync = false;  // zero the workspace's synchronisation words first
  const vt_emit* emit = nullptr;  // emit the quantised partial sums (fp16, persistent)
};

static vt_status decode_impl(const vt_shard_spec* spec, const WeightView& W, vt_kv_view* kv,
                             const vt_layer_io* io, int32_t pos, uint32_t phases, void* ws,
                             size_t ws_bytes, void* stream, const StackView& S = StackView());

static vt_status check_phases(const vt_shard_spec* spec, const vt_layer_io* io, uint32_t phases) {
  if (!spec || !io) return fail(VT_ERR_ARG, "null spec or io");
  if (phases & ~(VT_ATTN | VT_FFN | VT_STAGED | VT_COOPERATIVE))
    return fail(VT_ERR_ARG, "unknown phase bits 0x%x", phases);
  if (!(phases & (VT_ATTN | VT_FFN))) return fail(VT_ERR_ARG, "no phase selected");
  if ((phases & VT_STAGED) && (phases & VT_COOPERATIVE))
    return fail(VT_ERR_ARG, "VT_COOPERATIVE applies to the persistent launch, not VT_STAGED");
  return VT_OK;
}

extern "C" vt_status vt_layer_decode(const vt_shard_spec* spec, const vt_layer_weights* w,
                                     vt_kv_view* kv, const vt_layer_io* io, int32_t pos,
                                     uint32_t phases, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  return vt::layer_decode_ws(spec, w, kv, io, pos, phases, ws, ws_bytes, stream, false);
}

vt_status vt::layer_decode_ws(const vt_shard_spec* spec, const vt_layer_weights* w, vt_kv_view* kv,
                              const vt_layer_io* io, int32_t pos, uint32_t phases, void* ws,
                              size_t ws_bytes, void* stream, bool clear_sync) {
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
  StackView S;
  S.clear_sync = clear_sync;
  return decode_impl(spec, W, kv, io, pos, phases, ws, ws_bytes, stream, S);
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

extern "C" vt_status vt_layer_decode_emit(const vt_shard_spec* spec, const vt_layer_weights* w,
                                          vt_kv_view* kv, const vt_layer_io* io, int32_t pos,
                                          uint32_t phases, const vt_emit* emit, void* ws,
                                          size_t ws_bytes, void* stream) {
  clear_error();
  vt_status st = check_phases(spec, io, phases);
  if (st != VT_OK) return st;
  if (!emit) return fail(VT_ERR_ARG, "null emit description");
  if (phases & VT_STAGED) return fail(VT_ERR_UNSUPPORTED, "emission runs in the persistent launch only");
  if (spec->dims.hidden % 32) return fail(VT_ERR_UNSUPPORTED, "hidden %d is not a multiple of 32", spec->dims.hidden);
  auto msg = [&](const uint8_t* prec, const int32_t* off, const void* m, size_t bytes, bool on,
                 const char* name) -> vt_status {
    if (!m) return VT_OK;
    if (!on) return fail(VT_ERR_ARG, "%s message given but its phase does not run", name);
    if (!prec || !off) return fail(VT_ERR_ARG, "%s message without a plan", name);
    if (reinterpret_cast<uintptr_t>(off) % 4) return fail(VT_ERR_ALIGN, "%s offsets not 4-byte aligned", name);
    if (bytes >= static_cast<size_t>(kMaxBufferBytes))
      return fail(VT_ERR_UNSUPPORTED, "%s message of %zu bytes; at most 2 GiB", name, bytes);
    return VT_OK;
  };
  if ((st = msg(emit->prec_attn, emit->off_attn, emit->msg_attn, emit->msg_attn_bytes, phases & VT_ATTN,
                "attention")) != VT_OK)
    return st;
  if ((st = msg(emit->prec_ffn, emit->off_ffn, emit->msg_ffn, emit->msg_ffn_bytes, phases & VT_FFN, "FFN")) !=
      VT_OK)
    return st;
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
  StackView S;
  S.emit = emit;
  return decode_impl(spec, W, kv, io, pos, phases, ws, ws_bytes, stream, S);
}

extern "C" vt_status vt_stack_decode(const vt_shard_spec* spec, const vt_stack_weights* w,
                                     vt_kv_stack* kv, const vt_layer_io* io, int32_t pos, void* ws,
                                     size_t ws_bytes, void* stream) {
  clear_error();
  if (!spec || !w || !kv || !io) return fail(VT_ERR_ARG, "null spec, weights, KV or io");
  const int L = w->n_layers;
  if (L < 1 || L > 4096) return fail(VT_ERR_ARG, "n_layers %d outside 1..4096", L);
  if (kv->n_layers != L) return fail(VT_ERR_ARG, "KV stack has %d layers, weights %d", kv->n_layers, L);
  vt_status st = check_weights(*spec, &w->w, true, true);
  if (st != VT_OK) return st;
  if (!io->attn_partial || !io->h || !io->ffn_partial || !io->y)
    return fail(VT_ERR_ARG, "a stack needs attn_partial, h, ffn_partial and y ([n_layers][hidden] each)");
  const vt_layer_weights& w0 = w->w;
  const int64_t H = spec->dims.hidden, d = spec->dims.head_dim;
  const int64_t qd = static_cast<int64_t>(spec->info.n_q_heads) * d;
  const int64_t kd = static_cast<int64_t>(spec->info.n_kv_heads) * d;
  const int64_t F = spec->info.n_cols;
  // layer l's matrix at l * rows * ld elements past layer 0's (bytes below)
  const bool heads = spec->info.n_q_heads > 0, cols = F > 0;
  StackView S;
  S.n_layers = L;
  const int64_t rows[7] = {qd, kd, kd, H, F, F, H};
  const int64_t lds[7] = {w0.ld_q, w0.ld_k, w0.ld_v, w0.ld_o, w0.ld_g, w0.ld_u, w0.ld_d};
  const bool has[7] = {heads, heads, heads, heads, cols, cols, cols};
  for (int i = 0; i < 7; ++i) S.lst_w[i] = has[i] ? rows[i] * lds[i] * 2 : 0;
  S.lst_kv = static_cast<int64_t>(kv->n_kv_heads) * kv->capacity * kv->head_dim;
  vt_kv_view v0{kv->k, kv->v, kv->capacity, kv->n_kv_heads, kv->head_dim, kv->len};
  WeightView W{};
  W.fmt = dec::FMT_F16;
  W.g_attn = w0.g_attn;
  W.g_ffn = w0.g_ffn;
  const void* ptrs[7] = {w0.wq, w0.wk, w0.wv, w0.wo, w0.wg, w0.wu, w0.wd};
  for (int i = 0; i < 7; ++i) {
    W.w[i] = ptrs[i];
    W.ld[i] = lds[i] * 2;
  }
  st = decode_impl(spec, W, &v0, io, pos, VT_ATTN | VT_FFN, ws, ws_bytes, stream, S);
  if (st == VT_OK) kv->len = v0.len;
  return st;
}

static vt_status decode_impl(const vt_shard_spec* spec, const WeightView& W, vt_kv_view* kv,
                             const vt_layer_io* io, int32_t pos, uint32_t phases, void* ws,
                             size_t ws_bytes, void* stream, const StackView& S) {
  const bool attn = phases & VT_ATTN, ffn = phases & VT_FFN, staged = phases & VT_STAGED;
  const bool coop = phases & VT_COOPERATIVE;
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
  attn_chunking(D.head_dim, in.n_q_heads, attn ? pos - p_first : 0, di->cus, &P.cl, &P.nchunk);
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
  P.n_layers = S.n_layers;
  for (int i = 0; i < 7; ++i) P.lst_w[i] = S.lst_w[i];
  P.lst_kv = S.lst_kv;
  if (S.emit) {
    P.eprec_a = S.emit->prec_attn;
    P.eoff_a = S.emit->off_attn;
    P.emsg_a = static_cast<uint8_t*>(S.emit->msg_attn);
    P.emsg_a_bytes = static_cast<uint32_t>(S.emit->msg_attn_bytes);
    P.eprec_f = S.emit->prec_ffn;
    P.eoff_f = S.emit->off_ffn;
    P.emsg_f = static_cast<uint8_t*>(S.emit->msg_ffn);
    P.emsg_f_bytes = static_cast<uint32_t>(S.emit->msg_ffn_bytes);
  }

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
  // The grid barrier needs every workgroup resident at once: one per CU,
  // and the occupancy query confirms a CU holds at least one. A plain
  // launch is used (the cooperative launch API adds ~20 us per launch);
  // the barrier's bounded wait reports rather than hangs if another
  // kernel were to hold CUs.
  const bool stack = S.n_layers > 1;
  if (stack && (staged || W.fmt != dec::FMT_F16 || pb != dec::PH_QKV || pe != dec::PH_DOWN))
    return fail(VT_ERR_UNSUPPORTED, "a stack runs fp16 layers, all phases, one launch");
  const dec::DecodeKernel kern = stack    ? dec::decode_stack_kernel()
                                 : S.emit ? dec::decode_comm_kernel(pb, pe)
                                          : dec::decode_kernel_for(pb, pe, W.fmt);
  if (!staged) {
    int per_cu = 0;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, dec::NT, lds);
    if (e != hipSuccess) return fail(VT_ERR_HIP, "occupancy query: %s", hipGetErrorString(e));
    if (per_cu < 1)
      return fail(VT_ERR_UNSUPPORTED, "decode kernel does not fit on a CU with %zu bytes of LDS", lds);
  }
  // every check has passed: the launches below are the call's
  if (S.clear_sync) {
    const int nwords = static_cast<int>(L.qkv / 4);
    hipLaunchKernelGGL(dec::zero_words, dim3((nwords + 255) / 256), dim3(256), 0, s,
                       static_cast<uint32_t*>(ws), nwords);
    e = hipGetLastError();
    if (e != hipSuccess) return fail(VT_ERR_HIP, "workspace clear launch: %s", hipGetErrorString(e));
  }
  if (staged) {
    for (int ph = pb; ph <= pe && e == hipSuccess; ++ph) {
      P.phase_begin = P.phase_end = ph;
      hipLaunchKernelGGL(dec::decode_kernel_for(ph, ph, W.fmt), dim3(di->cus), dim3(dec::NT), lds, s, P);
      e = hipGetLastError();
    }
  } else {
    P.phase_begin = pb;
    P.phase_end = pe;
    if (coop) {
      void* args[] = {&P};
      e = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(kern), dim3(di->cus), dim3(dec::NT), args,
                                     static_cast<unsigned>(lds), s);
    } else {
      hipLaunchKernelGGL(kern, dim3(di->cus), dim3(dec::NT), lds, s, P);
      e = hipGetLastError();
    }
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
