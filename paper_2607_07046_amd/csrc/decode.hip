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

constexpr int NT = 512;          // threads per workgroup
constexpr int NW = NT / kWave;   // waves per workgroup
constexpr int SEG = 512;         // fp16 elements per piece (64 lanes x 8)
constexpr int PF = 16;           // pieces in flight per wave
constexpr int MAX_SLOTS = 4096;  // pieces per workgroup round (one float each)
constexpr int REC = 4;           // attention partial record = head_dim + REC floats
constexpr unsigned kSpinLimit = 1u << 20;  // about a second of polling

enum { PH_QKV = 0, PH_ATTN = 1, PH_O = 2, PH_GATEUP = 3, PH_DOWN = 4 };
enum { SW_BAR = 0, SW_EXIT = 1, SW_ERR = 2, SW_GROUP = 16 };

struct Params {
  int H, d, nq, nkv, G, ncols, pos, cap, nchunk, cl;
  float eps, rope_base;
  const uint16_t *g_attn, *wq, *wk, *wv, *wo, *g_ffn, *wg, *wu, *wd;
  int64_t ld_q, ld_k, ld_v, ld_o, ld_g, ld_u, ld_d;
  uint16_t *kc, *vc;
  const uint16_t *x, *peer_a, *peer_f;
  uint16_t *p_attn, *h, *p_ffn, *y;
  float *qkv, *part, *o, *m;
  unsigned* sync;
  int phase_begin, phase_end;
};

// ---------------------------------------------------------------------------
// grid barrier (only between phases of one persistent launch)
// ---------------------------------------------------------------------------
__device__ __forceinline__ void grid_arrive(unsigned* sync) {
  __syncthreads();
  if (threadIdx.x == 0) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    __hip_atomic_fetch_add(sync + SW_BAR, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

__device__ __forceinline__ void grid_wait(unsigned* sync, unsigned target) {
  if (threadIdx.x == 0) {
    unsigned n = 0;
    while (__hip_atomic_load(sync + SW_BAR, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
      __builtin_amdgcn_s_sleep(1);
      if (++n > kSpinLimit) {  // never expected: report instead of hanging
        sync_or(sync + SW_ERR, 1u);
        break;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// row sources: virtual row index -> address of its first element
// ---------------------------------------------------------------------------
struct RowsQKV {
  const uint16_t *wq, *wk, *wv;
  int64_t lq, lk, lv;
  int nqd, nkd;
  __device__ __forceinline__ const uint16_t* operator()(int r) const {
    if (r < nqd) return wq + static_cast<int64_t>(r) * lq;
    r -= nqd;
    if (r < nkd) return wk + static_cast<int64_t>(r) * lk;
    return wv + static_cast<int64_t>(r - nkd) * lv;
  }
};

struct RowsOne {
  const uint16_t* w;
  int64_t ld;
  __device__ __forceinline__ const uint16_t* operator()(int r) const {
    return w + static_cast<int64_t>(r) * ld;
  }
};

struct RowsPair {  // row 2j -> a[j], row 2j+1 -> b[j]
  const uint16_t *a, *b;
  int64_t la, lb;
  __device__ __forceinline__ const uint16_t* operator()(int r) const {
    return (r & 1) ? b + static_cast<int64_t>(r >> 1) * lb : a + static_cast<int64_t>(r >> 1) * la;
  }
};

template <class Rows>
__device__ __forceinline__ u32x4 fetch(const Rows& rows, int row0, int q, int nseg, int K, int lane) {
  const int lr = q / nseg;
  const int s = q - lr * nseg;
  const int col = s * SEG + lane * 8;
  u32x4 v = {0u, 0u, 0u, 0u};
  if (col < K) v = load_stream(rows(row0 + lr) + col);
  return v;
}

// Dot product of one piece with the staged input vector xs (zero beyond K).
__device__ __forceinline__ float dot_piece(const u32x4 w, const float* xs, int s, int K, int lane) {
  const int col = s * SEG + lane * 8;
  float f[8];
  unpack8(w, f);
  if (col + 8 > K) {  // tail piece: drop row padding, whatever it holds
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (col + e >= K) f[e] = 0.f;
  }
  const f32x4 a = *reinterpret_cast<const f32x4*>(xs + col);
  const f32x4 b = *reinterpret_cast<const f32x4*>(xs + col + 4);
  float r = f[0] * a.x;
  r = fmaf(f[1], a.y, r);
  r = fmaf(f[2], a.z, r);
  r = fmaf(f[3], a.w, r);
  r = fmaf(f[4], b.x, r);
  r = fmaf(f[5], b.y, r);
  r = fmaf(f[6], b.z, r);
  r = fmaf(f[7], b.w, r);
  return r;
}

// One GEMV phase over ``units`` output units of U virtual rows of K columns.
// ``stage`` waits for the phase's input and fills xs[0, nseg*SEG) (ending in
// a workgroup barrier); ``epi(unit, sums)`` consumes each unit's U dot
// products.
template <int U, class Rows, class Stage, class Epi>
__device__ __forceinline__ void gemv_phase(const Rows& rows, int units, int K, float* xs,
                                           float* slots, Stage stage, Epi epi) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int u0 = static_cast<int>(static_cast<int64_t>(units) * blockIdx.x / gridDim.x);
  const int u1 = static_cast<int>(static_cast<int64_t>(units) * (blockIdx.x + 1) / gridDim.x);
  const int nseg = (K + SEG - 1) / SEG;
  const int upr = nseg ? max(1, MAX_SLOTS / (U * nseg)) : max(1, u1 - u0);
  bool staged = false;
  int ua = u0;
  do {
    const int ub = min(u1, ua + upr);
    const int np = (ub - ua) * U * nseg;
    const int q0 = static_cast<int>(static_cast<int64_t>(np) * wave / NW);
    const int q1 = static_cast<int>(static_cast<int64_t>(np) * (wave + 1) / NW);
    const int row0 = ua * U;
    u32x4 buf[PF];
#pragma unroll
    for (int i = 0; i < PF; ++i)
      if (q0 + i < q1) buf[i] = fetch(rows, row0, q0 + i, nseg, K, lane);
    if (!staged) {
      stage();
      staged = true;
    }
    float acc = 0.f;
    for (int base = q0; base < q1; base += PF) {
#pragma unroll
      for (int i = 0; i < PF; ++i) {
        const int q = base + i;
        if (q < q1) {
          const u32x4 w = buf[i];
          if (q + PF < q1) buf[i] = fetch(rows, row0, q + PF, nseg, K, lane);
          const int s = q % nseg;
          acc += dot_piece(w, xs, s, K, lane);
          if (s == nseg - 1 || q == q1 - 1) {
            const float t = wave_sum(acc);
            if (lane == 0) slots[q] = t;
            acc = 0.f;
          } else if (lane == 0) {
            slots[q] = 0.f;
          }
        }
      }
    }
    __syncthreads();
    for (int lu = threadIdx.x; lu < ub - ua; lu += NT) {
      float v[U];
#pragma unroll
      for (int j = 0; j < U; ++j) {
        float a = 0.f;
        const float* sl = slots + (lu * U + j) * nseg;
        for (int s = 0; s < nseg; ++s) a += sl[s];
        v[j] = a;
      }
      epi(ua + lu, v);
    }
    __syncthreads();
    ua = ub;
  } while (ua < u1);
}

// xs[k] = v[k] * rstd * g[k] for k < n (v, g fp16), zero up to npad.
__device__ __forceinline__ void stage_rmsnorm(const uint16_t* v, const uint16_t* g, int n, int npad,
                                              float eps, float* xs, float* red) {
  float ss = 0.f;
  for (int k8 = threadIdx.x; k8 < n / 8; k8 += NT) {
    float f[8];
    unpack8(load16(v + k8 * 8), f);
#pragma unroll
    for (int e = 0; e < 8; ++e) ss = fmaf(f[e], f[e], ss);
  }
  ss = block_sum<NT>(ss, red);
  const float rstd = 1.0f / sqrtf(ss / static_cast<float>(n) + eps);
  for (int k8 = threadIdx.x; k8 < n / 8; k8 += NT) {
    float f[8], gg[8];
    unpack8(load16(v + k8 * 8), f);
    unpack8(load16(g + k8 * 8), gg);
#pragma unroll
    for (int e = 0; e < 8; ++e) xs[k8 * 8 + e] = f[e] * rstd * gg[e];
  }
  for (int k = n + threadIdx.x; k < npad; k += NT) xs[k] = 0.f;
  __syncthreads();
}

__device__ __forceinline__ void stage_copy(const float* v, int n, int npad, float* xs) {
  for (int k = threadIdx.x; k < npad; k += NT) xs[k] = k < n ? v[k] : 0.f;
  __syncthreads();
}

__host__ __device__ __forceinline__ int padded(int K) { return ((K + SEG - 1) / SEG) * SEG; }

// ---------------------------------------------------------------------------
// phase 1: attention over the shard's KV groups
// ---------------------------------------------------------------------------
__device__ __forceinline__ void phase_attn(const Params& P, float* lds, bool wait, unsigned target) {
  const int d = P.d, G = P.G, CL = P.cl;
  const int TPP = d / 8;               // threads per cached position
  const int t = threadIdx.x;
  const int pl = t / TPP;              // this thread's position within the chunk
  const int dc = (t % TPP) * 8;        // and its 8 dimensions
  const int items = P.nkv * P.nchunk;
  const float scale = 1.0f / sqrtf(static_cast<float>(d));
  // LDS layout (floats): qs[G*d] | S[G*CL] | Vs[CL*d] | kn[d] | vn[d] | flag
  float* qs = lds;
  float* S = qs + G * d;
  float* Vs = S + G * CL;
  float* kn = Vs + CL * d;
  float* vn = kn + d;
  int* flag = reinterpret_cast<int*>(vn + d);

  bool waited = false;
  for (int it = blockIdx.x;; it += gridDim.x) {
    const bool valid = it < items;
    const int g = valid ? it / P.nchunk : 0;
    const int c = valid ? it - g * P.nchunk : 0;
    const int p = c * CL + pl;
    // cached keys/values of this thread's position (data independent of phase 0)
    u32x4 kreg = {0u, 0u, 0u, 0u}, vreg = {0u, 0u, 0u, 0u};
    if (valid && p < P.pos) {
      const int64_t off = (static_cast<int64_t>(g) * P.cap + p) * d + dc;
      kreg = load16(P.kc + off);
      vreg = load16(P.vc + off);
    }
    if (!waited) {
      if (wait) grid_wait(P.sync, target);
      waited = true;
    }
    if (!valid) break;

    // rotated, pre-scaled queries of the group's G heads
    const int half = d / 2;
    for (int idx = t; idx < G * half; idx += NT) {
      const int jj = idx / half, i = idx - jj * half;
      const float* q = P.qkv + static_cast<int64_t>(g * G + jj) * d;
      float c0, s0;
      rope_angle(P.pos, i, d, P.rope_base, c0, s0);
      const float a = q[2 * i], b = q[2 * i + 1];
      qs[jj * d + 2 * i] = (a * c0 - b * s0) * scale;
      qs[jj * d + 2 * i + 1] = (a * s0 + b * c0) * scale;
    }
    const bool has_new = (P.pos >= c * CL) && (P.pos < (c + 1) * CL);
    if (has_new) {  // this item appends the new token's key and value
      const float* kq = P.qkv + static_cast<int64_t>(P.nq) * d + static_cast<int64_t>(g) * d;
      const float* vq = P.qkv + static_cast<int64_t>(P.nq + P.nkv) * d + static_cast<int64_t>(g) * d;
      const int64_t slot = (static_cast<int64_t>(g) * P.cap + P.pos) * d;
      for (int i = t; i < half; i += NT) {
        float c0, s0;
        rope_angle(P.pos, i, d, P.rope_base, c0, s0);
        const float a = kq[2 * i], b = kq[2 * i + 1];
        const uint16_t k0 = f2h(a * c0 - b * s0), k1 = f2h(a * s0 + b * c0);
        kn[2 * i] = h2f(k0);
        kn[2 * i + 1] = h2f(k1);
        P.kc[slot + 2 * i] = k0;
        P.kc[slot + 2 * i + 1] = k1;
      }
      for (int i = t; i < d; i += NT) {
        const uint16_t v0 = f2h(vq[i]);
        vn[i] = h2f(v0);
        P.vc[slot + i] = v0;
      }
    }
    __syncthreads();

    // scores of this thread's position for each of the G heads
    float kf[8];
    if (p == P.pos) {
#pragma unroll
      for (int e = 0; e < 8; ++e) kf[e] = kn[dc + e];
    } else {
      unpack8(kreg, kf);
    }
    const bool live = p <= P.pos && pl < CL;
    for (int jj = 0; jj < G; ++jj) {
      const float* qq = qs + jj * d + dc;
      float sacc = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) sacc = fmaf(qq[e], kf[e], sacc);
      sacc = group_sum(sacc, TPP);
      if ((t % TPP) == 0 && pl < CL) S[jj * CL + pl] = live ? sacc : -INFINITY;
    }
    // stage values (fp32) for the weighted sum
    if (pl < CL) {
      float vf[8];
      if (p == P.pos) {
#pragma unroll
        for (int e = 0; e < 8; ++e) vf[e] = vn[dc + e];
      } else if (p < P.pos) {
        unpack8(vreg, vf);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) vf[e] = 0.f;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) Vs[pl * d + dc + e] = vf[e];
    }
    __syncthreads();

    // softmax statistics of the chunk, one wave per head
    const int wave = t / kWave, lane = t % kWave;
    float* rec0 = P.part + (static_cast<int64_t>(g) * P.nchunk + c) * G * (d + REC);
    for (int jj = wave; jj < G; jj += NW) {
      const float s = lane < CL ? S[jj * CL + lane] : -INFINITY;
      const float mx = wave_max(s);
      const float e = (lane < CL && s != -INFINITY) ? __expf(s - mx) : 0.f;
      const float l = wave_sum(e);
      if (lane < CL) S[jj * CL + lane] = e;
      if (lane == 0) {
        rec0[jj * (d + REC) + d] = mx;
        rec0[jj * (d + REC) + d + 1] = l;
      }
    }
    __syncthreads();
    // unnormalised weighted sum of values
    for (int idx = t; idx < G * d; idx += NT) {
      const int jj = idx / d, dd = idx - jj * d;
      float a = 0.f;
      for (int q = 0; q < CL; ++q) a = fmaf(S[jj * CL + q], Vs[q * d + dd], a);
      rec0[jj * (d + REC) + dd] = a;
    }
    // the last chunk of group g to finish merges the group's chunks
    __syncthreads();
    if (t == 0) {
      const unsigned old = __hip_atomic_fetch_add(P.sync + SW_GROUP + g, 1u, __ATOMIC_ACQ_REL,
                                                  __HIP_MEMORY_SCOPE_AGENT);
      *flag = (old == static_cast<unsigned>(P.nchunk - 1));
    }
    __syncthreads();
    if (*flag) {
      const float* recg = P.part + static_cast<int64_t>(g) * P.nchunk * G * (d + REC);
      for (int idx = t; idx < G * d; idx += NT) {
        const int jj = idx / d, dd = idx - jj * d;
        float M = -INFINITY;
        for (int cc = 0; cc < P.nchunk; ++cc) M = fmaxf(M, recg[(cc * G + jj) * (d + REC) + d]);
        float L = 0.f, a = 0.f;
        for (int cc = 0; cc < P.nchunk; ++cc) {
          const float* r = recg + (cc * G + jj) * (d + REC);
          const float w = __expf(r[d] - M);
          L = fmaf(r[d + 1], w, L);
          a = fmaf(r[dd], w, a);
        }
        P.o[static_cast<int64_t>(g * G + jj) * d + dd] = a / L;
      }
      __syncthreads();
      if (t == 0) sync_store(P.sync + SW_GROUP + g, 0u);
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// the kernel
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(NT) decode_kernel(Params P) {
  extern __shared__ float lds[];
  // LDS: xs / attention scratch (aliased) | slots[MAX_SLOTS] | red[NW]
  const int kmax = max(max(padded(P.H), padded(P.nq * P.d)), padded(P.ncols));
  const int attn = P.G * P.d + P.G * P.cl + P.cl * P.d + 2 * P.d + 4;
  float* xs = lds;
  float* slots = lds + max(kmax, attn);
  float* red = slots + MAX_SLOTS;

  for (int ph = P.phase_begin; ph <= P.phase_end; ++ph) {
    const bool wait = ph > P.phase_begin;
    const unsigned target = static_cast<unsigned>(ph - P.phase_begin) * gridDim.x;
    auto waitfor = [&]() {
      if (wait) grid_wait(P.sync, target);
    };
    switch (ph) {
      case PH_QKV: {
        RowsQKV rows{P.wq, P.wk, P.wv, P.ld_q, P.ld_k, P.ld_v, P.nq * P.d, P.nkv * P.d};
        gemv_phase<1>(
            rows, (P.nq + 2 * P.nkv) * P.d, P.H, xs, slots,
            [&]() {
              waitfor();
              stage_rmsnorm(P.x, P.g_attn, P.H, padded(P.H), P.eps, xs, red);
            },
            [&](int r, const float* v) { P.qkv[r] = v[0]; });
        break;
      }
      case PH_ATTN:
        phase_attn(P, lds, wait, target);
        break;
      case PH_O: {
        RowsOne rows{P.wo, P.ld_o};
        const int K = P.nq * P.d;
        gemv_phase<1>(
            rows, P.H, K, xs, slots,
            [&]() {
              waitfor();
              stage_copy(P.o, K, padded(K), xs);
            },
            [&](int r, const float* v) {
              const float pa = v[0];
              P.p_attn[r] = f2h(pa);
              const float hv = h2f(P.x[r]) + pa + (P.peer_a ? h2f(P.peer_a[r]) : 0.f);
              P.h[r] = f2h(hv);
            });
        break;
      }
      case PH_GATEUP: {
        RowsPair rows{P.wg, P.wu, P.ld_g, P.ld_u};
        gemv_phase<2>(
            rows, P.ncols, P.H, xs, slots,
            [&]() {
              waitfor();
              stage_rmsnorm(P.h, P.g_ffn, P.H, padded(P.H), P.eps, xs, red);
            },
            [&](int j, const float* v) {
              const float gt = v[0], up = v[1];
              P.m[j] = gt / (1.0f + __expf(-gt)) * up;
            });
        break;
      }
      case PH_DOWN: {
        RowsOne rows{P.wd, P.ld_d};
        const int K = P.ncols;
        gemv_phase<1>(
            rows, P.H, K, xs, slots,
            [&]() {
              waitfor();
              stage_copy(P.m, K, padded(K), xs);
            },
            [&](int r, const float* v) {
              const float pf = v[0];
              P.p_ffn[r] = f2h(pf);
              if (P.y) P.y[r] = f2h(h2f(P.h[r]) + pf + (P.peer_f ? h2f(P.peer_f[r]) : 0.f));
            });
        break;
      }
    }
    if (ph < P.phase_end) grid_arrive(P.sync);
  }
  if (P.phase_end > P.phase_begin) {  // the last workgroup out clears the barrier words
    __syncthreads();
    if (threadIdx.x == 0) {
      const unsigned old = __hip_atomic_fetch_add(P.sync + SW_EXIT, 1u, __ATOMIC_ACQ_REL,
                                                  __HIP_MEMORY_SCOPE_AGENT);
      if (old == gridDim.x - 1) {
        sync_store(P.sync + SW_BAR, 0u);
        sync_store(P.sync + SW_EXIT, 0u);
      }
    }
  }
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
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(dec::decode_kernel),
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              static_cast<int>(di.max_lds));
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
  size_t sync, qkv, part, o, m, total;
};

static int attn_chunk(int d) { return dec::NT / (d / 8); }

static DecodeWs decode_ws_layout(const vt_shard_spec& s, int32_t max_ctx) {
  const vt_shard_info& in = s.info;
  const int d = s.dims.head_dim;
  const int G = s.dims.n_heads / s.dims.n_kv_heads;
  const int64_t nchunk = (max_ctx + attn_chunk(d) - 1) / attn_chunk(d);
  DecodeWs w{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off += static_cast<size_t>(round_up(static_cast<int64_t>(bytes), 256));
    return at;
  };
  w.sync = take(sizeof(unsigned) * (dec::SW_GROUP + in.n_kv_heads + 16));
  w.qkv = take(sizeof(float) * (in.n_q_heads + 2 * in.n_kv_heads) * d);
  w.part = take(sizeof(float) * in.n_kv_heads * nchunk * G * (d + dec::REC));
  w.o = take(sizeof(float) * in.n_q_heads * d);
  w.m = take(sizeof(float) * (in.n_cols + 8));
  w.total = off;
  return w;
}

size_t decode_workspace_bytes(const vt_shard_spec& s, int32_t max_ctx) {
  return decode_ws_layout(s, max_ctx).total;
}

vt_status check_weights(const vt_shard_spec& s, const vt_layer_weights* w, bool attn, bool ffn) {
  if (!w) return fail(VT_ERR_ARG, "null weights");
  const int H = s.dims.hidden, d = s.dims.head_dim;
  const vt_shard_info& in = s.info;
  auto mat = [&](const void* p, int64_t ld, int64_t rowlen, const char* name) -> vt_status {
    if (!p) return fail(VT_ERR_ARG, "weight %s is NULL", name);
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
      if ((st = mat(w->wq, w->ld_q, H, "wq")) != VT_OK) return st;
      if ((st = mat(w->wk, w->ld_k, H, "wk")) != VT_OK) return st;
      if ((st = mat(w->wv, w->ld_v, H, "wv")) != VT_OK) return st;
      if ((st = mat(w->wo, w->ld_o, static_cast<int64_t>(in.n_q_heads) * d, "wo")) != VT_OK)
        return st;
    }
  }
  if (ffn) {
    if ((st = gain(w->g_ffn, "g_ffn")) != VT_OK) return st;
    if (in.n_cols > 0) {
      if ((st = mat(w->wg, w->ld_g, H, "wg")) != VT_OK) return st;
      if ((st = mat(w->wu, w->ld_u, H, "wu")) != VT_OK) return st;
      if ((st = mat(w->wd, w->ld_d, in.n_cols, "wd")) != VT_OK) return st;
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

extern "C" vt_status vt_layer_decode(const vt_shard_spec* spec, const vt_layer_weights* w,
                                     vt_kv_view* kv, const vt_layer_io* io, int32_t pos,
                                     uint32_t phases, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  if (!spec || !io) return fail(VT_ERR_ARG, "null spec or io");
  if (phases & ~(VT_ATTN | VT_FFN | VT_STAGED)) return fail(VT_ERR_ARG, "unknown phase bits 0x%x", phases);
  const bool attn = phases & VT_ATTN, ffn = phases & VT_FFN, staged = phases & VT_STAGED;
  if (!attn && !ffn) return fail(VT_ERR_ARG, "no phase selected");
  const vt_layer_dims& D = spec->dims;
  const vt_shard_info& in = spec->info;
  vt_status st = check_weights(*spec, w, attn, ffn);
  if (st != VT_OK) return st;
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
  P.cap = kv ? kv->capacity : 0;
  P.cl = attn_chunk(D.head_dim);
  P.nchunk = (ctx + P.cl - 1) / P.cl;
  P.eps = D.rms_eps;
  P.rope_base = D.rope_base;
  P.g_attn = static_cast<const uint16_t*>(w->g_attn);
  P.wq = static_cast<const uint16_t*>(w->wq);
  P.wk = static_cast<const uint16_t*>(w->wk);
  P.wv = static_cast<const uint16_t*>(w->wv);
  P.wo = static_cast<const uint16_t*>(w->wo);
  P.g_ffn = static_cast<const uint16_t*>(w->g_ffn);
  P.wg = static_cast<const uint16_t*>(w->wg);
  P.wu = static_cast<const uint16_t*>(w->wu);
  P.wd = static_cast<const uint16_t*>(w->wd);
  P.ld_q = w->ld_q;
  P.ld_k = w->ld_k;
  P.ld_v = w->ld_v;
  P.ld_o = w->ld_o;
  P.ld_g = w->ld_g;
  P.ld_u = w->ld_u;
  P.ld_d = w->ld_d;
  P.kc = kv ? static_cast<uint16_t*>(kv->k) : nullptr;
  P.vc = kv ? static_cast<uint16_t*>(kv->v) : nullptr;
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

  const int kmax = std::max({dec::padded(P.H), dec::padded(P.nq * P.d),
                             dec::padded(P.ncols)});
  const int attn_f = P.G * P.d + P.G * P.cl + P.cl * P.d + 2 * P.d + 4;
  const size_t lds = sizeof(float) * (std::max(kmax, attn_f) + dec::MAX_SLOTS + dec::NW);
  if (lds > di->max_lds)
    return fail(VT_ERR_UNSUPPORTED, "shape needs %zu bytes of LDS, device has %zu", lds, di->max_lds);

  const int pb = attn ? dec::PH_QKV : dec::PH_GATEUP;
  const int pe = ffn ? dec::PH_DOWN : dec::PH_O;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipSuccess;
  if (staged) {
    for (int ph = pb; ph <= pe && e == hipSuccess; ++ph) {
      P.phase_begin = P.phase_end = ph;
      hipLaunchKernelGGL(dec::decode_kernel, dim3(di->cus), dim3(dec::NT), lds, s, P);
      e = hipGetLastError();
    }
  } else {
    P.phase_begin = pb;
    P.phase_end = pe;
    void* args[] = {&P};
    e = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(dec::decode_kernel), dim3(di->cus),
                                   dim3(dec::NT), args, static_cast<unsigned>(lds), s);
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
