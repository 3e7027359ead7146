// cmsd.hip - gfx950 kernels and C ABI for the logit pass of confidence-modulated
// speculative decoding (arXiv 2508.15371, Sec. III.B).  Interface: include/cmsd.h.
//
// Kernels (all bandwidth-bound streaming reductions; no MFMA):
//   k_confidence    one workgroup (64/128/256 threads, by launch shape) per drafter
//                   row: single streaming pass with an online max / sum-exp /
//                   sum(e*(z-m)) reduction, top-1 and top-2 tracking at chunk
//                   granularity, DPP wave reductions, LDS only for the cross-wave
//                   combine; epilogue forms H, margins and C (optionally the
//                   variance of the logits).
//   k_draft_len     one workgroup: per-sequence mean confidence, clipped floor,
//                   exclusive scan of k_b + 1 into packed target-row offsets.
//   k_target_rows   one workgroup per packed target row: max / sum-exp of the row,
//                   scalar (ballot + s_bcnt1) count of logits above the drafted
//                   token's, the acceptance decision of that position, and the
//                   row's slot in the workspace.
//   k_final_parts   one wave per (sequence, vocabulary slice): first rejection from
//                   the row slots (ballot; in cmsd_logit_pass the draft length and
//                   accept tests too), then fp64 slice partials of the residual (or
//                   bonus) row.
//   k_final_sample  one workgroup per sequence: slice scan, then an exact in-slice
//                   inverse-CDF locate that repeats the scan's sums bit for bit.
//   k_row_pass      cmsd_logit_pass's row pass: drafter rows (as k_confidence) and
//                   dense target rows (as k_target_rows, decisions deferred) in one
//                   grid.
//   k_pass_decide   cmsd_logit_pass on large launches and in GREEDY mode, one wave
//                   per sequence: draft length, accept tests and first rejection,
//                   written once for the final kernels (GREEDY: the final outputs).
//   k_fused_pass    cmsd_logit_pass_fused, one launch for small batches: the row pass,
//                   then the last row workgroup of each sequence (atomic count behind
//                   a device fence) decides and samples with the same functions.
//   k_draft_parts / k_draft_pick   the same slice machinery for one softmax sample
//                   per drafter row.
//
// Compile-time tuning knobs (defaults are the measured best on gfx950): CMSD_STREAM_DEPTH
// and CMSD_DEEP_DEPTH (row-pass rounds of loads in flight for short and long launches),
// CMSD_KEEP_MAX_ROUND (64-thread drafter rows keep
// their max round in registers), CMSD_SLICE_UNITS and CMSD_SUB_PER_WG (final-token slice
// size and slices per one-wave workgroup).
//
// Numerics: exponentials are evaluated as 2^(z*log2e - m*log2e) with one FMA and
// v_exp_f32; per-thread partial sums are fp32 over 32-element chunks, the
// cross-thread combines and every decision-side formula are fp64.  Reductions have
// a fixed order, so results are bit-reproducible run to run.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#include <atomic>
#include <mutex>
#include <type_traits>

#include "cmsd.h"

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr double kLn2 = 0.69314718055994530942;
// Finite "minus infinity" for the scaled running max, and the finite value a drafter
// row's -inf logits are clamped to before their normaliser and entropy terms: its
// scaled value (kMaskedLogit*log2e) lies below kNegBig, so a chunk of masked logits
// never raises the running max, and z*log2e - ms stays finite for every logit with
// |z| < 2^96, so a masked logit adds exactly 0 to both sums.
constexpr float kNegBig = -0x1p126f;
constexpr float kMaskedLogit = -0x1p127f;

// ----------------------------------------------------------------------------- logit element types
struct Bf16 { uint16_t bits; };

template <typename T> struct Elem;
template <> struct Elem<float> {
  static constexpr int VEC = 4;   // elements per 16-byte vector
  static constexpr int U = 8;     // vectors per thread per chunk (32 elements)
  static constexpr uint32_t NINF = 0xff800000u;  // -inf, as one element's bits
  __device__ static float load(const float* p) { return *p; }
  // n < VEC elements at p as one raw 16-byte vector, padded with -inf
  __device__ static uint4 raw_partial(const float* p, int n) {
    uint4 r;
    r.x = n > 0 ? __float_as_uint(p[0]) : NINF;
    r.y = n > 1 ? __float_as_uint(p[1]) : NINF;
    r.z = n > 2 ? __float_as_uint(p[2]) : NINF;
    r.w = n > 3 ? __float_as_uint(p[3]) : NINF;
    return r;
  }
  __device__ static uint4 raw_ninf() { return make_uint4(NINF, NINF, NINF, NINF); }
  __device__ static void unpack(const uint4& v, float* f) {
    f[0] = __uint_as_float(v.x); f[1] = __uint_as_float(v.y);
    f[2] = __uint_as_float(v.z); f[3] = __uint_as_float(v.w);
  }
  // -inf (and only values below kMaskedLogit, outside the logit range) to kMaskedLogit:
  // an unsigned min on the raw bits, since negative floats order by magnitude there
  __device__ static uint32_t clamp_word(uint32_t w) { return w < 0xff000000u ? w : 0xff000000u; }
  // the clamp value (kMaskedLogit) in every element: padding that adds exactly 0 to the sums
  __device__ static uint4 raw_masked() { return make_uint4(0xff000000u, 0xff000000u, 0xff000000u, 0xff000000u); }
  __device__ static uint4 clamp_masked(const uint4& v) {
    return make_uint4(clamp_word(v.x), clamp_word(v.y), clamp_word(v.z), clamp_word(v.w));
  }
};
template <> struct Elem<Bf16> {
  static constexpr int VEC = 8;
  static constexpr int U = 4;     // 32 elements per chunk
  static constexpr uint32_t NINF = 0xff80u;
  __device__ static float load(const Bf16* p) { return __uint_as_float(uint32_t(p->bits) << 16); }
  __device__ static uint4 raw_partial(const Bf16* p, int n) {
    uint32_t h[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) h[e] = e < n ? uint32_t(p[e].bits) : NINF;
    return make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
  }
  __device__ static uint4 raw_ninf() {
    const uint32_t w = NINF | (NINF << 16);
    return make_uint4(w, w, w, w);
  }
  __device__ static void unpack(const uint4& v, float* f) {
    f[0] = __uint_as_float(v.x << 16); f[1] = __uint_as_float(v.x & 0xffff0000u);
    f[2] = __uint_as_float(v.y << 16); f[3] = __uint_as_float(v.y & 0xffff0000u);
    f[4] = __uint_as_float(v.z << 16); f[5] = __uint_as_float(v.z & 0xffff0000u);
    f[6] = __uint_as_float(v.w << 16); f[7] = __uint_as_float(v.w & 0xffff0000u);
  }
  // -inf (0xff80) to kMaskedLogit (0xff00) in both halves of a word at once: a packed
  // unsigned 16-bit min (v_pk_min_u16), one instruction per two logits
  typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
  __device__ static uint32_t clamp_word(uint32_t w) {
    const u16x2 lim = {0xff00, 0xff00};
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_min(__builtin_bit_cast(u16x2, w), lim));
  }
  // the clamp value (kMaskedLogit) in every element: padding that adds exactly 0 to the sums
  __device__ static uint4 raw_masked() { return make_uint4(0xff00ff00u, 0xff00ff00u, 0xff00ff00u, 0xff00ff00u); }
  __device__ static uint4 clamp_masked(const uint4& v) {
    return make_uint4(clamp_word(v.x), clamp_word(v.y), clamp_word(v.z), clamp_word(v.w));
  }
};

// Whether a stream of raw 16-byte vectors held a -inf logit, for the drafter-row flag
// (the clamped values no longer show it).  bf16: the matrix core sums each vector's
// eight logits against ones (one MFMA per vector, beside the VALU work); a -inf
// anywhere makes the sums -inf, and with |z| < 2^96 no finite sum overflows.  The
// sums of one lane's data land in other lanes, so the answer is taken over the wave.
// fp32: the unsigned max of the raw bits reaches 0xff800000 only for -inf.
template <typename T> struct MaskProbe;
template <> struct MaskProbe<Bf16> {
  typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
  typedef float f32x4 __attribute__((ext_vector_type(4)));
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  __device__ void add(const uint4& v) {
    const uint4 ones = make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, v), __builtin_bit_cast(bf16x8, ones),
                                                  acc, 0, 0, 0);
  }
  __device__ bool hit() const {
    return !(acc[0] > -INFINITY && acc[1] > -INFINITY && acc[2] > -INFINITY && acc[3] > -INFINITY);
  }
};
template <> struct MaskProbe<float> {
  uint32_t m = 0;
  __device__ void add(const uint4& v) {
    const uint32_t a = v.x > v.y ? v.x : v.y, b = v.z > v.w ? v.z : v.w;
    m = m > a ? m : a;
    m = m > b ? m : b;
  }
  __device__ bool hit() const { return m >= 0xff800000u; }
};

// Row geometry: `head` leading elements before the first 16-byte boundary, `nvec`
// aligned 16-byte vectors, `tail` trailing elements.
struct Geom {
  int head;
  int tail;
  int64_t nvec;
};

template <typename T>
__device__ __forceinline__ Geom row_geom(const T* row, int64_t V) {
  constexpr int VEC = Elem<T>::VEC;
  const int mis = int(reinterpret_cast<uintptr_t>(row) & 15u);
  int64_t head = mis ? (16 - mis) / int(sizeof(T)) : 0;
  if (head > V) head = V;
  const int64_t rest = V - head;
  Geom g;
  g.head = int(head);
  g.nvec = rest / VEC;
  g.tail = int(rest - g.nvec * VEC);
  return g;
}

__device__ __forceinline__ float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Streaming 16-byte load with the nontemporal hint: logit rows are read once per
// pass, and the hint keeps them from displacing reused lines in the caches.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld_stream(const uint4* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// ----------------------------------------------------------------------------- wave / block reductions
// Wave64 all-reduce: DPP quad permutes and row mirrors inside each 16-lane row,
// then the four row results are combined through readlane (uniform result).
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) { return __int_as_float(dpp_i<CTRL>(__float_as_int(v))); }
template <int CTRL>
__device__ __forceinline__ double dpp_d(double v) {
  return __hiloint2double(dpp_i<CTRL>(__double2hiint(v)), dpp_i<CTRL>(__double2loint(v)));
}
__device__ __forceinline__ float rl_f(float v, int l) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l)); }
__device__ __forceinline__ double rl_d(double v, int l) {
  return __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(v), l),
                          __builtin_amdgcn_readlane(__double2loint(v), l));
}

struct OpMax { __device__ float operator()(float a, float b) const { return fmaxf(a, b); } };
struct OpSumD { __device__ double operator()(double a, double b) const { return a + b; } };
struct OpSumI { __device__ int operator()(int a, int b) const { return a + b; } };
struct OpMinI { __device__ int operator()(int a, int b) const { return a < b ? a : b; } };
struct OpMaxI { __device__ int operator()(int a, int b) const { return a > b ? a : b; } };

template <typename Op>
__device__ __forceinline__ float wave_all_f(float v, Op op) {
  v = op(v, dpp_f<0xB1>(v));   // quad_perm [1,0,3,2]
  v = op(v, dpp_f<0x4E>(v));   // quad_perm [2,3,0,1]
  v = op(v, dpp_f<0x141>(v));  // row_half_mirror
  v = op(v, dpp_f<0x140>(v));  // row_mirror
  return op(op(rl_f(v, 0), rl_f(v, 16)), op(rl_f(v, 32), rl_f(v, 48)));
}
template <typename Op>
__device__ __forceinline__ double wave_all_d(double v, Op op) {
  v = op(v, dpp_d<0xB1>(v));
  v = op(v, dpp_d<0x4E>(v));
  v = op(v, dpp_d<0x141>(v));
  v = op(v, dpp_d<0x140>(v));
  return op(op(rl_d(v, 0), rl_d(v, 16)), op(rl_d(v, 32), rl_d(v, 48)));
}
template <typename Op>
__device__ __forceinline__ int wave_all_i(int v, Op op) {
  v = op(v, dpp_i<0xB1>(v));
  v = op(v, dpp_i<0x4E>(v));
  v = op(v, dpp_i<0x141>(v));
  v = op(v, dpp_i<0x140>(v));
  return op(op(__builtin_amdgcn_readlane(v, 0), __builtin_amdgcn_readlane(v, 16)),
            op(__builtin_amdgcn_readlane(v, 32), __builtin_amdgcn_readlane(v, 48)));
}

// Block all-reduce through LDS: one slot per wave, combined in wave order by every
// thread (so every thread holds the same, order-fixed result).  `slot` must hold
// BD/64 elements; the leading barrier protects the slot from a previous use.
template <int BD, typename Op>
__device__ __forceinline__ float block_all_f(float v, Op op, float* slot) {
  constexpr int NW = BD / 64;
  const float w = wave_all_f(v, op);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) slot[threadIdx.x >> 6] = w;
  __syncthreads();
  float r = slot[0];
#pragma unroll
  for (int i = 1; i < NW; ++i) r = op(r, slot[i]);
  return r;
}
template <int BD, typename Op>
__device__ __forceinline__ double block_all_d(double v, Op op, double* slot) {
  constexpr int NW = BD / 64;
  const double w = wave_all_d(v, op);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) slot[threadIdx.x >> 6] = w;
  __syncthreads();
  double r = slot[0];
#pragma unroll
  for (int i = 1; i < NW; ++i) r = op(r, slot[i]);
  return r;
}
template <int BD, typename Op>
__device__ __forceinline__ int block_all_i(int v, Op op, int* slot) {
  constexpr int NW = BD / 64;
  const int w = wave_all_i(v, op);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) slot[threadIdx.x >> 6] = w;
  __syncthreads();
  int r = slot[0];
#pragma unroll
  for (int i = 1; i < NW; ++i) r = op(r, slot[i]);
  return r;
}

// Block sums of N doubles in one LDS round: every thread receives all N totals
// (waves combined in order).  `lds` must hold N * BD/64 doubles.
template <int BD, int N>
__device__ __forceinline__ void block_sum_n(double (&v)[N], double* lds) {
  constexpr int NW = BD / 64;
  double w[N];
#pragma unroll
  for (int j = 0; j < N; ++j) w[j] = wave_all_d(v[j], OpSumD());
  __syncthreads();
  if ((threadIdx.x & 63) == 0) {
#pragma unroll
    for (int j = 0; j < N; ++j) lds[j * NW + (threadIdx.x >> 6)] = w[j];
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < N; ++j) {
    double r = lds[j * NW];
    for (int i = 1; i < NW; ++i) r += lds[j * NW + i];
    v[j] = r;
  }
}

// Streams the nr full rounds of a row: round k is U vectors per thread at
// vp[(k*U + u)*BD + t].  DEPTH rounds of loads are kept in flight in a ring of
// registers (fully unrolled, so each slot is consumed and then refilled in place:
// no register copies).  The main loop covers the rounds whose refills all exist, so
// no load there sits behind a branch: the number of loads in flight is the same on
// every path, and the wait before a round covers that round only while the later
// rounds stay in flight.  The last rounds (fewer than 2*DEPTH) follow with guarded
// refills; the first DEPTH are always requested.  prep() runs once the first loads
// are issued (work that must precede the first round overlaps their latency);
// consume(raw[U], k) is called in round order.
#ifndef CMSD_STREAM_DEPTH
#define CMSD_STREAM_DEPTH 2
#endif
template <int U, int BD, int DEPTH, typename P, typename F>
__device__ __forceinline__ void stream_rounds(const uint4* vp, int64_t nr, int t, P&& prep, F&& consume) {
  if (nr <= 0) {
    prep();
    return;
  }
  // the first DEPTH rounds, issued unconditionally (a row of fewer rounds reads vp[0],
  // the same 16 bytes for every lane, in their place)
  uint4 buf[DEPTH][U];
#pragma unroll
  for (int d = 0; d < DEPTH; ++d) {
#pragma unroll
    for (int u = 0; u < U; ++u) buf[d][u] = ld_stream(vp + (d < nr ? ((int64_t)d * U + u) * BD + t : 0));
    __builtin_amdgcn_sched_barrier(0);  // rounds leave in order, as the loop refills them
  }
  prep();
  int64_t k0 = 0;
  for (; k0 + 2 * DEPTH <= nr; k0 += DEPTH) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) {
      const int64_t k = k0 + d;
      consume(buf[d], k);
      const int64_t kn = k + DEPTH;
#pragma unroll
      for (int u = 0; u < U; ++u) buf[d][u] = ld_stream(vp + (kn * U + u) * BD + t);
      __builtin_amdgcn_sched_barrier(0);  // the refill leaves before the next round is consumed
    }
  }
  for (; k0 < nr; k0 += DEPTH) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) {
      const int64_t k = k0 + d;
      if (k < nr) {
        consume(buf[d], k);
        const int64_t kn = k + DEPTH;
        if (kn < nr) {
#pragma unroll
          for (int u = 0; u < U; ++u) buf[d][u] = ld_stream(vp + (kn * U + u) * BD + t);
        }
      }
    }
  }
}

// ----------------------------------------------------------------------------- streaming row state
// Online normaliser in base-2 units relative to a running scaled max ms = fl(max*log2e):
//   A = sum 2^x,  T = sum 2^x * x,  x = z*log2e - ms.
// When ms grows by -d (d <= 0) the partial sums rescale as A' = 2^d A and
// T' = 2^d (T + d A).  T becomes NaN exactly when the row holds a -inf logit
// (0 * -inf); that case is redone with a guarded pass in the epilogue.
struct NormState {
  float ms = kNegBig;
  float A = 0.f;
  float T = 0.f;
};

template <int N, bool GUARD, bool WITH_T>
__device__ __forceinline__ void norm_chunk(NormState& s, const float* f, uint32_t valid, float cmax) {
  const float ms_new = fmaxf(s.ms, cmax * kLog2e);
  const float d = s.ms - ms_new;
  const float sc = fexp2(d);
  float cs = 0.f, ct = 0.f;
#pragma unroll
  for (int j = 0; j < N; ++j) {
    float x = fmaf(f[j], kLog2e, -ms_new);
    float e = fexp2(x);
    if (GUARD) {
      const bool ok = (valid >> j) & 1u;
      e = ok ? e : 0.f;
      x = ok ? x : 0.f;
    }
    cs += e;
    if (WITH_T) ct = fmaf(e, x, ct);
  }
  if (WITH_T) s.T = fmaf(sc, fmaf(d, s.A, s.T), ct);
  s.A = fmaf(s.A, sc, cs);
  s.ms = ms_new;
}

template <int N>
__device__ __forceinline__ float chunk_max(const float* f) {
  float m = f[0];
#pragma unroll
  for (int j = 1; j < N; ++j) m = fmaxf(m, f[j]);
  return m;
}

// Drafter-row state: normaliser plus the top-2 of chunk maxima and the first chunk
// (in this thread's index order) that attains the thread's maximum.
// With the logit variance: count, mean and centred second moment of this thread's
// elements, merged chunk by chunk (Chan et al.'s pairwise update), so no sum of
// squares of raw logits is ever formed.  A -inf element turns them into NaN; that
// case is redone with the guarded pass.
struct ConfState {
  NormState n;
  float t1 = -INFINITY;
  float t2 = -INFINITY;
  int gid = -1;
  float vn = 0.f, vmean = 0.f, vm2 = 0.f;
};

template <int N, bool GUARD>
__device__ __forceinline__ void var_chunk(ConfState& s, const float* f, uint32_t valid) {
  float cs = 0.f;
  int cnt = N;
  if (GUARD) cnt = __popc(valid);
#pragma unroll
  for (int j = 0; j < N; ++j) cs += (!GUARD || ((valid >> j) & 1u)) ? f[j] : 0.f;
  if (cnt == 0) return;
  const float cm = GUARD ? cs / (float)cnt : cs * (1.f / (float)N);
  float c2 = 0.f;
#pragma unroll
  for (int j = 0; j < N; ++j) {
    const float d = (!GUARD || ((valid >> j) & 1u)) ? f[j] - cm : 0.f;
    c2 = fmaf(d, d, c2);
  }
  const float n1 = s.vn + (float)cnt;
  const float delta = cm - s.vmean;
  const float w = (float)cnt / n1;
  s.vmean = fmaf(delta, w, s.vmean);
  s.vm2 = s.vm2 + c2 + delta * delta * (s.vn * w);
  s.vn = n1;
}

template <int N, bool GUARD, bool VAR>
__device__ __forceinline__ void conf_chunk(ConfState& s, const float* f, uint32_t valid, int cid) {
  const float cmax = chunk_max<N>(f);
  s.gid = cmax > s.t1 ? cid : s.gid;
  s.t2 = __builtin_amdgcn_fmed3f(s.t1, s.t2, cmax);
  s.t1 = fmaxf(s.t1, cmax);
  norm_chunk<N, GUARD, true>(s.n, f, valid, cmax);
  if (VAR) var_chunk<N, GUARD>(s, f, valid);
}

template <bool VAR>
__device__ __forceinline__ void conf_one(ConfState& s, float z, int cid) {
  float f[1] = {z};
  conf_chunk<1, false, VAR>(s, f, 1u, cid);
}

// Enumerates the elements of one chunk of thread t (chunk ids: 0 head element,
// 1..nr full rounds, nr+1 the partial round, nr+2 the tail element) and returns the
// lowest index holding `m` plus the largest other value in that chunk.
template <typename T, int BD>
__device__ void rescan_chunk(const T* row, const Geom& g, int64_t nr, int cid, float m, int64_t& idx, float& other) {
  using E = Elem<T>;
  constexpr int VEC = E::VEC, U = E::U;
  const int t = threadIdx.x;
  idx = INT64_MAX;
  other = -INFINITY;
  auto visit = [&](int64_t i, float z) {
    if (idx == INT64_MAX && z == m) idx = i;
    else other = fmaxf(other, z);
  };
  if (cid == 0) {
    if (t < g.head) visit(t, E::load(row + t));
  } else if (cid == nr + 2) {
    const int64_t base = g.head + g.nvec * VEC;
    if (t < g.tail) visit(base + t, E::load(row + base + t));
  } else if (cid >= 1 && cid <= nr + 1) {
    const uint4* vp = reinterpret_cast<const uint4*>(row + g.head);
    for (int u = 0; u < U; ++u) {
      const int64_t j = (int64_t)(cid - 1) * U * BD + (int64_t)u * BD + t;
      if (j < g.nvec) {
        float f[VEC];
        E::unpack(vp[j], f);
        for (int e = 0; e < VEC; ++e) visit(g.head + j * VEC + e, f[e]);
      }
    }
  }
}

// ----------------------------------------------------------------------------- K1 confidence
struct ConfArgs {
  float l_ent, l_margin, l_soft, beta_m;
  double inv_lnV;   // 1 / ln(vocab)
  double inv_soft;  // 1 / (1 - 1/vocab), the softmax margin's normaliser
};

// The drafter-row record from the row's reductions: max m, second value z2 (the
// largest value other than the first occurrence of m; -inf with one finite logit),
// A = sum 2^(z log2e - m log2e) and T = sum of 2^x x over the same terms.
__device__ __forceinline__ cmsd_row_stats row_stats_record(float m, float z2, double A, double Tsum, uint32_t flags,
                                                           int top1, const ConfArgs& a) {
  // one fp64 division per row (1/A) and one for the sigmoid; the per-call constants come
  // as reciprocals, so the row's wave spends little time on this dependent chain
  const double invA = 1.0 / A;
  const double Tn = Tsum * kLn2;
  double H = (double)log1pf((float)(A - 1.0)) - Tn * invA;  // ln A = log1p(A - 1), A - 1 exact in fp64
  H = H < 0.0 ? 0.0 : H;
  const double dm = (double)m, dz2 = (double)z2;
  const double margin = z2 == -INFINITY ? INFINITY : dm - dz2;
  const double msoft = z2 == -INFINITY ? invA : (double)(-expm1f((float)(dz2 - dm))) * invA;
  const double c_ent = 1.0 - H * a.inv_lnV;
  const double tm = (double)a.beta_m * margin;
  const double c_m = tm == INFINITY ? 1.0 : 1.0 / (1.0 + (double)expf((float)-tm));
  const double c_s = fmin(1.0, msoft * a.inv_soft);
  const double C = (double)a.l_ent * c_ent + (double)a.l_margin * c_m + (double)a.l_soft * c_s;
  cmsd_row_stats o;
  o.max_logit = m;
  o.sum_exp = (float)A;
  o.entropy = (float)H;
  o.margin_soft = (float)msoft;
  o.margin_logit = (float)margin;
  o.conf = (float)C;
  o.top1 = top1;
  o.flags = flags;
  return o;
}

// One drafter row -> its stats record (and, with VAR, its logit variance), by one
// workgroup of BD threads.  KEEP_WIDE keeps the max round's vectors in registers for
// every workgroup size, not only 64-thread rows (the kernel's registers permitting).
#ifndef CMSD_KEEP_MAX_ROUND
#define CMSD_KEEP_MAX_ROUND 1
#endif
template <typename T, int BD, bool VAR, int DEPTH = CMSD_STREAM_DEPTH, bool KEEP_WIDE = false>
__device__ __forceinline__ void conf_row(const T* __restrict__ row, int64_t V, const ConfArgs& a,
                                         cmsd_row_stats* __restrict__ out, float* __restrict__ var_out) {
  using E = Elem<T>;
  constexpr bool KEEP = CMSD_KEEP_MAX_ROUND && (BD == 64 || KEEP_WIDE);
  constexpr int VEC = E::VEC, U = E::U, N = VEC * U;
  constexpr int ND = VAR ? 5 : 2;  // fp64 sums of the epilogue: A, T (+ count, S1, S2)
  __shared__ double sd[(VAR ? 3 : 1) * (BD / 64)];
  __shared__ float sf[BD / 64];
  __shared__ double ep_d[ND][BD / 64];
  __shared__ float ep_f[2][BD / 64];
  __shared__ int ep_i[3][BD / 64];
  const int t = threadIdx.x;
  {
    const Geom g = row_geom(row, V);
    const uint4* vp = reinterpret_cast<const uint4*>(row + g.head);
    const int64_t per_round = (int64_t)U * BD;
    const int64_t nr = g.nvec / per_round;

    ConfState s;
    // KEEP: the vectors of the round that set this thread's maximum stay in registers,
    // so the epilogue finds the max index without reading that round again
    uint4 keep[KEEP ? U : 1];
#pragma unroll
    for (int u = 0; u < (KEEP ? U : 1); ++u) keep[u] = make_uint4(0u, 0u, 0u, 0u);
    // Masked (-inf) logits: every logit is clamped to at least kMaskedLogit before the
    // sums (a masked one then adds exactly 0 to A and T), and a probe over the raw
    // vectors (plus a test of the single head, tail and partial-round elements) records
    // that the row held one: one read of every row.  Only the variance moments of a
    // masked row are redone, without its -inf logits, by a second pass.
    MaskProbe<T> probe;
    bool ninf_el = false;
    auto clamp1 = [&](float z) {
      ninf_el |= z == -INFINITY;
      return fmaxf(z, kMaskedLogit);
    };

    // full rounds, next round's loads issued before the current one is consumed
    // the head elements are loaded and folded in once the first rounds are requested
    stream_rounds<U, BD, DEPTH>(vp, nr, t, [&] {
      if (t < g.head) conf_one<VAR>(s, clamp1(E::load(row + t)), 0);
    }, [&](const uint4 (&raw)[U], int64_t k) {
      float f[N];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        probe.add(raw[u]);
        E::unpack(E::clamp_masked(raw[u]), f + u * VEC);
      }
      conf_chunk<N, false, VAR>(s, f, 0xffffffffu, int(k + 1));
      if (KEEP) {
        const bool up = s.gid == int(k + 1);
#pragma unroll
        for (int u = 0; u < (KEEP ? U : 1); ++u) {
          keep[u].x = up ? raw[u].x : keep[u].x;
          keep[u].y = up ? raw[u].y : keep[u].y;
          keep[u].z = up ? raw[u].z : keep[u].z;
          keep[u].w = up ? raw[u].w : keep[u].w;
        }
      }
    });
    // partial round: whole vectors clamped and probed as in the full rounds; lanes past
    // the row show the probe zeros and hold the clamp value, which adds exactly 0 to A
    // and T as a masked logit does, so the round takes the unguarded arithmetic (the
    // variance moments, which must not see padding, keep the guarded form and -inf)
    const int64_t rb = nr * per_round;
    if (rb < g.nvec) {
      float f[N];
      uint32_t valid = 0;
      uint4 pv[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t j = rb + (int64_t)u * BD + t;
        pv[u] = make_uint4(0u, 0u, 0u, 0u);
        if (j < g.nvec) {
          pv[u] = ld_stream(vp + j);
          valid |= ((1u << VEC) - 1u) << (u * VEC);
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        probe.add(pv[u]);
        const bool in = (valid >> (u * VEC)) & 1u;
        E::unpack(in ? E::clamp_masked(pv[u]) : (VAR ? E::raw_ninf() : E::raw_masked()), f + u * VEC);
      }
      conf_chunk<N, VAR, VAR>(s, f, valid, int(nr + 1));
    }
    const int64_t tail0 = g.head + g.nvec * VEC;
    if (t < g.tail) conf_one<VAR>(s, clamp1(E::load(row + tail0 + t)), int(nr + 2));

    // ---- epilogue: row max, first index of the max, second logit, normaliser
    const float m = block_all_f<BD>(s.t1, OpMax(), sf);
    const float ms_row = m * kLog2e;
    const float d = s.n.ms - ms_row;
    const float sc = fexp2(d);
    const double Ad = (double)(s.n.A * sc);
    const double Td = (double)(sc * fmaf(d, s.n.A, s.n.T));
    const bool is_max = s.t1 == m;
    int64_t idx = INT64_MAX;
    float other = -INFINITY;
    if (is_max) {
      if (KEEP && s.gid >= 1 && s.gid <= nr) {
#pragma unroll
        for (int u = 0; u < (KEEP ? U : 1); ++u) {
          float fv[VEC];
          E::unpack(keep[u], fv);
          const int64_t j = (int64_t)(s.gid - 1) * U * BD + (int64_t)u * BD + t;
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            if (idx == INT64_MAX && fv[e] == m) idx = g.head + j * VEC + e;
            else other = fmaxf(other, fv[e]);
          }
        }
      } else {
        rescan_chunk<T, BD>(row, g, nr, s.gid, m, idx, other);
      }
    }
    const float contrib = is_max ? s.t2 : s.t1;
    const int idx32 = idx == INT64_MAX ? INT32_MAX : int(idx);

    // one LDS round for: sum A, sum T, max of the other chunk maxima, number of
    // threads holding the max, the lowest max index with its chunk's other value, and
    // whether the row held a -inf logit
    double A, Tsum, vN = 0.0, vS1 = 0.0, vS2 = 0.0;
    float cmx, s_oth;
    int nmax, top1, ninf = 0;
    {
      const double wA = wave_all_d(Ad, OpSumD());
      const double wT = wave_all_d(Td, OpSumD());
      // variance moments about the row max: n, n (mean - m), M2 + n (mean - m)^2
      double wN = 0.0, wS1 = 0.0, wS2 = 0.0;
      if (VAR) {
        const double n = (double)s.vn, dmu = (double)s.vmean - (double)m;
        wN = wave_all_d(n, OpSumD());
        wS1 = wave_all_d(n * dmu, OpSumD());
        wS2 = wave_all_d(s.vn > 0.f ? (double)s.vm2 + n * dmu * dmu : 0.0, OpSumD());
      }
      const float wc = wave_all_f(contrib, OpMax());
      const int wn = wave_all_i(is_max ? 1 : 0, OpSumI());
      const int wi = wave_all_i(idx32, OpMinI());
      const unsigned long long own = __ballot(idx32 == wi && is_max);
      const float wo = own ? rl_f(other, __builtin_ctzll(own)) : -INFINITY;
      const int wninf = __ballot(ninf_el || probe.hit()) != 0ull ? 1 : 0;
      __syncthreads();
      if ((t & 63) == 0) {
        const int w = t >> 6;
        ep_d[0][w] = wA;
        ep_d[1][w] = wT;
        if constexpr (VAR) {
          ep_d[ND - 3][w] = wN;
          ep_d[ND - 2][w] = wS1;
          ep_d[ND - 1][w] = wS2;
        }
        ep_f[0][w] = wc;
        ep_f[1][w] = wo;
        ep_i[0][w] = wn;
        ep_i[1][w] = wi;
        ep_i[2][w] = wninf;
      }
      __syncthreads();
      A = ep_d[0][0];
      Tsum = ep_d[1][0];
      cmx = ep_f[0][0];
      s_oth = ep_f[1][0];
      nmax = ep_i[0][0];
      top1 = ep_i[1][0];
      ninf = ep_i[2][0];
      if constexpr (VAR) {
        vN = ep_d[ND - 3][0];
        vS1 = ep_d[ND - 2][0];
        vS2 = ep_d[ND - 1][0];
      }
#pragma unroll
      for (int w = 1; w < BD / 64; ++w) {
        A += ep_d[0][w];
        Tsum += ep_d[1][w];
        if constexpr (VAR) {
          vN += ep_d[ND - 3][w];
          vS1 += ep_d[ND - 2][w];
          vS2 += ep_d[ND - 1][w];
        }
        cmx = fmaxf(cmx, ep_f[0][w]);
        nmax += ep_i[0][w];
        ninf |= ep_i[2][w];
        if (ep_i[1][w] < top1) {
          top1 = ep_i[1][w];
          s_oth = ep_f[1][w];
        }
      }
    }
    const uint32_t flags = ninf ? 1u : 0u;  // bit 0: the row holds -inf logits
    if (VAR && ninf) {
      // the variance moments of a masked row, about the row max and without its -inf
      // logits (the clamped values entered the streaming moments)
      double vm[3] = {0.0, 0.0, 0.0};
      auto acc = [&](float z) {
        if (z > -INFINITY) {
          const double dz = (double)z - (double)m;
          vm[0] += 1.0;
          vm[1] += dz;
          vm[2] += dz * dz;
        }
      };
      if (t < g.head) acc(E::load(row + t));
      for (int64_t j = t; j < g.nvec; j += BD) {
        float f[VEC];
        E::unpack(vp[j], f);
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc(f[e]);
      }
      if (t < g.tail) acc(E::load(row + tail0 + t));
      block_sum_n<BD, 3>(vm, sd);
      vN = vm[0];
      vS1 = vm[1];
      vS2 = vm[2];
    }
    __syncthreads();
    if (t == 0) {
      // a second value at kMaskedLogit or below is a clamped -inf: the row has one finite logit
      const float z2 = nmax >= 2 ? m : fmaxf(cmx, s_oth);
      *out = row_stats_record(m, z2 <= kMaskedLogit ? -INFINITY : z2, A, Tsum, flags, top1, a);
      if (VAR) {
        const double v = (vS2 - vS1 * (vS1 / vN)) / vN;
        *var_out = (float)(v > 0.0 ? v : 0.0);
      }
    }
    __syncthreads();
  }
}

template <typename T, int BD, bool VAR, int DEPTH>
__global__ __launch_bounds__(BD) void k_confidence(const T* __restrict__ logits, int64_t n_rows, int64_t V,
                                                   int64_t stride, ConfArgs a, cmsd_row_stats* __restrict__ out,
                                                   float* __restrict__ var_out) {
  for (int64_t r = blockIdx.x; r < n_rows; r += gridDim.x)
    conf_row<T, BD, VAR, DEPTH>(logits + r * stride, V, a, out + r, VAR ? var_out + r : nullptr);
}

// ----------------------------------------------------------------------------- K2 draft length
// One workgroup.  The confidences of a tile of sequences are read with coalesced loads
// (consecutive threads, consecutive records) into LDS, padded to k_max + 1 floats per
// sequence so the per-sequence reads hit distinct banks; thread b then sums its
// sequence left to right in fp64, clips the floor, and a block scan of k_b + 1 gives
// the offsets.
constexpr int kDraftBD = 1024;
constexpr int kDraftLds = 16384;  // staged confidences (64 KB)

__global__ __launch_bounds__(kDraftBD) void k_draft_len(const cmsd_row_stats* __restrict__ stats, int B, int k_min,
                                                        int k_max, float alpha, int32_t* __restrict__ k_out,
                                                        int32_t* __restrict__ off_out) {
  __shared__ float s_c[kDraftLds];
  __shared__ int s_w[kDraftBD / 64];
  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  const int ld = k_max + 1;                                  // LDS floats per sequence
  const int tile = kDraftLds / ld < kDraftBD ? kDraftLds / ld : kDraftBD;  // >= 3 (k_max <= 4096)
  int carry = 0;
  for (int base = 0; base < B; base += tile) {
    const int nb = B - base < tile ? B - base : tile;
    const int n = nb * k_max;
    const cmsd_row_stats* p = stats + (int64_t)base * k_max;
    for (int j0 = 0; j0 < n; j0 += 8 * kDraftBD) {          // 8 loads in flight per thread
      float c[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int j = j0 + u * kDraftBD + t;
        c[u] = j < n ? p[j].conf : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int j = j0 + u * kDraftBD + t;
        if (j < n) s_c[(j / k_max) * ld + j % k_max] = c[u];
      }
    }
    __syncthreads();
    int kb = 0;
    if (t < nb) {
      const float* q = s_c + t * ld;
      double sum = 0.0;
      for (int i = 0; i < k_max; ++i) sum += (double)q[i];
      const double x = (double)alpha * (sum / (double)k_max) * (double)k_max;
      const double fl = floor(x);
      kb = fl < (double)k_min ? k_min : (fl > (double)k_max ? k_max : (int)fl);
      k_out[base + t] = kb;
    }
    // exclusive scan of (k_b + 1) over the tile: wave scan by shuffles, then wave totals
    const int v = t < nb ? kb + 1 : 0;
    int incl = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int up = __shfl_up(incl, o);
      if (lane >= o) incl += up;
    }
    if (lane == 63) s_w[w] = incl;
    __syncthreads();
    int wpre = 0, tot = 0;
    for (int i = 0; i < kDraftBD / 64; ++i) {
      if (i < w) wpre += s_w[i];
      tot += s_w[i];
    }
    if (t < nb) off_out[base + t] = carry + wpre + incl - v;
    carry += tot;
    __syncthreads();  // s_c and s_w are refilled by the next tile
  }
  if (t == 0) off_out[B] = carry;
}

// ----------------------------------------------------------------------------- K3 target rows
struct VerifyArgs {
  const void* draft;
  int64_t dstride;
  const cmsd_row_stats* dstats;
  const void* target;
  int64_t tstride;
  int64_t target_rows;
  const int32_t* off;
  const int32_t* klen;
  const int32_t* drafted;
  const float* unif;
  int B;
  int k_max;
  int64_t V;
  int mode;
  int beta;
  float tau_base;
  float gamma;
  cmsd_target_stats* tstats;
  int32_t* n_acc;
  int32_t* next_tok;
  struct RowSlot* slots;  // workspace: [B][k_max+1], by sequence and position
  // the single-call pass (cmsd_logit_pass): dense rows, draft length and decisions made
  // from the row results by the final-token kernels
  struct PassSlot* pslots;  // workspace: [B][k_max+1]
  cmsd_row_stats* dstats_out;
  ConfArgs ca;
  int32_t* klen_out;
  int k_min;
  float alpha;
  int adaptive;
};

// Target-row results of the single-call pass by (sequence, position): everything the
// accept test of the position needs from the target row.
struct PassSlot {
  double A;       // sum 2^(z log2e - m log2e) of the row
  float m;        // row max
  float gz, zd;   // target and drafter logits of the drafted token
  int32_t ngt;    // logits above gz seen (wave counts stop once one reaches top_beta)
  int32_t top1;   // lowest index of the row max (GREEDY mode), else -1
  int32_t st;     // 1 drafted position, -1 the row after the last draft, -2 invalid drafted id
};

// Target-row results by (sequence, position), so the final-token pass reads a whole
// sequence's rows in one round trip.  `r` tags the packed row that wrote the slot.
struct RowSlot {
  float m;
  float A;
  int32_t acc;
  int32_t r;
  int32_t top1;  // lowest index of the row max (GREEDY mode), else -1
  float dm, dA;  // the drafter row's max and normaliser at this position (drafted positions)
  int32_t pad;
};

struct TargetState {
  NormState n;
  float t1 = -INFINITY;
  int gid = -1;  // first chunk (this thread's index order) attaining t1
};

template <int N, bool GUARD>
__device__ __forceinline__ void target_chunk(TargetState& s, const float* f, uint32_t valid, int cid, bool count,
                                             float gz, int beta, int& wcnt) {
  const float cmax = chunk_max<N>(f);
  s.gid = cmax > s.t1 ? cid : s.gid;
  s.t1 = fmaxf(s.t1, cmax);
  norm_chunk<N, GUARD, false>(s.n, f, valid, cmax);
  // wave-uniform: count only when the gate needs it, skip chunks where no lane holds
  // a logit above the drafted one, and stop once this wave alone has seen top_beta
  if (count && wcnt < beta && __ballot(cmax > gz) != 0ull) {
#pragma unroll
    for (int j = 0; j < N; ++j) wcnt += __popcll(__ballot(f[j] > gz));
  }
}

// The target row pass.  prep() resolves the drafted token (and with it `count` and
// `gz`) while the first rounds of the row are already in flight.
template <typename T, int BD, int DEPTH, typename P>
__device__ __forceinline__ void target_stream(const T* row, const Geom& g, const bool& count, const float& gz,
                                              int beta, TargetState& s, int& wcnt, P&& prep) {
  using E = Elem<T>;
  constexpr int VEC = E::VEC, U = E::U, N = VEC * U;
  const int t = threadIdx.x;
  const uint4* vp = reinterpret_cast<const uint4*>(row + g.head);
  const int64_t per_round = (int64_t)U * BD;
  const int64_t nr = g.nvec / per_round;
  stream_rounds<U, BD, DEPTH>(
      vp, nr, t,
      [&] {
        // the head element is requested with the rounds, before prep() waits for
        // its own loads (every lane loads, lanes past the head element 0)
        const float hv = E::load(row + (t < g.head ? t : 0));
        prep();
        float f[1] = {t < g.head ? hv : -INFINITY};
        target_chunk<1, true>(s, f, t < g.head ? 1u : 0u, 0, count, gz, beta, wcnt);
      },
      [&](const uint4 (&raw)[U], int64_t k) {
        float f[N];
#pragma unroll
        for (int u = 0; u < U; ++u) E::unpack(raw[u], f + u * VEC);
        target_chunk<N, false>(s, f, 0xffffffffu, int(k + 1), count, gz, beta, wcnt);
      });
  const int64_t rb = nr * per_round;
  if (rb < g.nvec) {
    float f[N];
    uint32_t valid = 0;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t j = rb + (int64_t)u * BD + t;
      if (j < g.nvec) {
        E::unpack(ld_stream(vp + j), f + u * VEC);
        valid |= ((1u << VEC) - 1u) << (u * VEC);
      } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) f[u * VEC + e] = -INFINITY;
      }
    }
    target_chunk<N, true>(s, f, valid, int(nr + 1), count, gz, beta, wcnt);
  }
  {
    const int64_t tail0 = g.head + g.nvec * VEC;
    float f[1] = {t < g.tail ? E::load(row + tail0 + t) : -INFINITY};
    target_chunk<1, true>(s, f, t < g.tail ? 1u : 0u, int(nr + 2), count, gz, beta, wcnt);
  }
}

// The accept test of one drafted position y: standard speculative sampling
// u < p_t(y) / p_d(y) in logs and fp64 (Sec. III.A), or in CM mode the
// confidence-modulated gate: fewer than top_beta target logits above z_t[y] and
// gap m_t - z_t[y] <= tau_base + gamma (1 - C) (Sec. III.B(c)).  GREEDY mode accepts
// the target's top token, or what the gate passes.  `count` says whether the gate's
// rank count was taken; *ng receives the reported count.
__device__ __forceinline__ int accept_test(int mode, int beta, float tau_base, float gamma, bool count, int ngt,
                                           float gz, float zd, float m, double A, float dm, float dA, float cm,
                                           float u, int yd, int top1, int* ng) {
  const double lpt = gz == -INFINITY ? -INFINITY : ((double)gz - (double)m) - log(A);
  const double lpd = zd == -INFINITY ? -INFINITY : ((double)zd - (double)dm) - log((double)dA);
  bool stoch;
  if (lpt == -INFINITY) stoch = false;
  else if (u == 0.f || lpd == -INFINITY) stoch = true;
  else stoch = log((double)u) < lpt - lpd;
  *ng = count ? (ngt < beta ? ngt : beta) : 0;
  const double gap = gz == -INFINITY ? INFINITY : (double)m - (double)gz;
  const double tau = (double)tau_base + (double)gamma * (1.0 - (double)cm);
  const bool gate = count && ngt < beta && gap <= tau;
  if (mode == CMSD_MODE_GREEDY) return (yd == top1 || gate) ? 1 : 0;  // the paper's rule, relaxed by the gate
  return (stoch || (mode == CMSD_MODE_CM && gate)) ? 1 : 0;
}

// One target row.  PASS = false: position q = i*B + b of cmsd_verify's grid over
// (sequence, position); the sequence's draft length and offsets and the position's
// drafted id and drafter stats are loaded in one round from q alone, positions past
// k_b (and sequences with an invalid length or offsets, which the final-token kernels
// report) end there, else the row is packed row off[b] + i and its accept test is made
// here.  PASS = true: dense row q = b*(k_max+1) + i of the single-call pass, whose
// accept test waits for the drafter stats (PassSlot).
template <typename T, int BD, bool PASS, int DEPTH = CMSD_STREAM_DEPTH>
__device__ __forceinline__ void target_row(const VerifyArgs& a, int64_t q) {
  using E = Elem<T>;
  __shared__ double sd[BD / 64];
  __shared__ float sf[BD / 64];
  __shared__ int si[BD / 64];
  const int t = threadIdx.x;
  // cmsd_verify's grid is position-major (q = i*B + b): every sequence's scored rows
  // (i <= k_b) come before the positions past the shorter drafts, whose workgroups only
  // read the draft length and exit; the single-call pass numbers its dense rows b*(k_max+1)+i
  const int b = PASS ? int(q / (a.k_max + 1)) : int(q % a.B);
  const int i = PASS ? int(q - (int64_t)b * (a.k_max + 1)) : int(q / a.B);
  const bool in_k = i < a.k_max;
  const int64_t drow = (int64_t)b * a.k_max + (in_k ? i : 0);
  int64_t r = q;
  int kb = a.k_max, y = -1;
  cmsd_row_stats ds{};
  if (!PASS) {
    if (b >= a.B) return;
    kb = a.klen[b];
    const int64_t ob = a.off[b], ob1 = a.off[b + 1];
    y = in_k ? a.drafted[drow] : -1;
    if (in_k) ds = a.dstats[drow];
    if (kb < 0 || kb > a.k_max || i > kb || ob < 0 || ob1 != ob + kb + 1 || ob1 > a.target_rows) return;
    r = ob + i;
  }
  const T* trow = reinterpret_cast<const T*>(a.target) + r * a.tstride;
  const Geom g = row_geom(trow, a.V);

  // The drafted token's target and drafter logits (the accept test and the rank count
  // need them): requested before the row's first rounds when the id is already known
  // (cmsd_verify), so their latency hides behind the rounds'; in the single-call pass
  // the id load itself waits for the first rounds to be requested (prep()).
  bool valid = true, has_draft = false, count = false;
  const bool layout = true;
  int yd = -1;
  float gz = -INFINITY, zd = -INFINITY, cm = 0.f, dm = 0.f, dA = 1.f;
  auto gather = [&] {
    if (has_draft) {
      yd = y;
      if (y < 0 || (int64_t)y >= a.V) {
        valid = false;
        has_draft = false;
      } else {
        gz = E::load(trow + y);
        zd = E::load(reinterpret_cast<const T*>(a.draft) + drow * a.dstride + y);
      }
    }
    count = has_draft && a.mode != CMSD_MODE_STANDARD && a.beta > 0;
  };
  if (!PASS) {
    has_draft = i < kb;
    cm = ds.conf;
    dm = ds.max_logit;
    dA = ds.sum_exp;
    gather();
  }
  auto prep = [&] {
    if (PASS) {
      has_draft = in_k;
      if (has_draft) y = a.drafted[drow];
      gather();
    }
  };
  TargetState s;
  int wcnt = 0;
  target_stream<T, BD, DEPTH>(trow, g, count, gz, a.beta, s, wcnt, prep);

  const float m = block_all_f<BD>(s.t1, OpMax(), sf);
  const float ms_row = m * kLog2e;
  const float sc = fexp2(s.n.ms - ms_row);
  int top1 = -1;
  if (a.mode == CMSD_MODE_GREEDY) {
    // lowest index of the row max: each thread holding it rescans its first such chunk
    int64_t idx = INT64_MAX;
    float other;
    if (s.t1 == m) {
      constexpr int U = Elem<T>::U;
      rescan_chunk<T, BD>(trow, g, g.nvec / ((int64_t)U * BD), s.gid, m, idx, other);
    }
    top1 = block_all_i<BD>(idx == INT64_MAX ? INT32_MAX : int(idx), OpMinI(), si);
  }
  double A;
  int ngt;
  {
    const double wA = wave_all_d((double)(s.n.A * sc), OpSumD());
    __syncthreads();
    if ((t & 63) == 0) {
      sd[t >> 6] = wA;
      si[t >> 6] = wcnt;
    }
    __syncthreads();
    A = sd[0];
    ngt = si[0];
#pragma unroll
    for (int w = 1; w < BD / 64; ++w) {
      A += sd[w];
      ngt += si[w];
    }
  }
  if (t == 0 && PASS) {
    a.pslots[r] = PassSlot{A, m, gz, zd, ngt, top1, !valid ? -2 : (has_draft ? 1 : -1)};
  } else if (t == 0) {
    cmsd_target_stats res{};
    res.max_logit = m;
    res.sum_exp = (float)A;
    res.top1 = top1;
    if (!valid) {
      res = cmsd_target_stats{NAN, NAN, -1, -2, -1, {0, 0, 0}};
    } else if (!has_draft) {
      res.n_greater = -1;
      res.accept = -1;
    } else {
      const float u = a.mode == CMSD_MODE_GREEDY ? 0.f : a.unif[r];
      res.accept = accept_test(a.mode, a.beta, a.tau_base, a.gamma, count, ngt, gz, zd, m, A, dm, dA, cm, u, yd,
                               top1, &res.n_greater);
    }
    a.tstats[r] = res;
    if (layout) a.slots[(int64_t)b * (a.k_max + 1) + i] = RowSlot{m, (float)A, res.accept, (int32_t)r, top1, dm, dA, 0};
  }
}

template <typename T, int BD, int DEPTH>
__global__ __launch_bounds__(BD) void k_target_rows(VerifyArgs a) {
  target_row<T, BD, false, DEPTH>(a, blockIdx.x);
}

// The row pass of cmsd_logit_pass: drafter rows (stats) and dense target rows in one
// grid, drafter rows first; the two kinds of row do not depend on each other.  Its
// bf16 drafter rows keep their max round in registers at every workgroup size when two
// rounds are in flight: 118 instead of 115 registers at 256 threads, still 4 waves per
// SIMD, and no re-read of that round before the record (64 sequences of 8 drafts: at
// V = 50257, 43.2 -> 42.6 us per step; at V = 152064, 78.3 -> 77.8).  Three rounds in
// flight, or fp32's 8-vector rounds, would lose a wave per SIMD.
template <typename T, int DEPTH>
constexpr bool kKeepWide = std::is_same<T, Bf16>::value && DEPTH == 2;
template <typename T, int BD, int DEPTH>
__global__ __launch_bounds__(BD) void k_row_pass(VerifyArgs a) {
  const int64_t nd = (int64_t)a.B * a.k_max;
  const int64_t r = blockIdx.x;
  if (r < nd)
    conf_row<T, BD, false, DEPTH, kKeepWide<T, DEPTH>>(reinterpret_cast<const T*>(a.draft) + r * a.dstride, a.V,
                                                         a.ca, a.dstats_out + r, nullptr);
  else
    target_row<T, BD, true, DEPTH>(a, r - nd);
}

// ----------------------------------------------------------------------------- K4 final token
// The final token of sequence b is an inverse-CDF sample over one target row (the
// bonus row k_b when every draft passed) or over the residual max(0, p_t - p_d) of
// the target and drafter rows at the first rejection c.  Two kernels:
//   k_final_parts   B x S one-wave workgroups, each covering one slice of the row
//                   (pair): fp64 partials {sum e_t, sum e_d, sum q0, sum_{q0>0} e_d}
//                   per slice, e = 2^(z log2e - m log2e), q0 = max(0, e_t - rho0 e_d)
//                   with rho0 = A_t / A_d from the row passes.
//   k_final_sample  one workgroup per sequence: rho = sum e_t / sum e_d from the
//                   fresh sums, slice masses corrected to first order in rho - rho0,
//                   a scan over slices, then an exact scan/locate inside one slice.
// A unit is the head (unit 0), one 16-byte vector (1..nvec) or the tail (nvec+1) of
// the target row, always handled as one raw 16-byte vector padded with -inf (whose
// weights are exactly 0); slices are runs of kSliceUnits units.  Small slices and
// one-wave partial groups keep every stage of this latency-bound pass short.
#ifndef CMSD_SLICE_UNITS
#define CMSD_SLICE_UNITS 256
#endif
constexpr int kPartBD = 64;  // one wave per slice group
constexpr int kSliceUnits = CMSD_SLICE_UNITS;
#ifndef CMSD_SUB_PER_WG
#define CMSD_SUB_PER_WG 1
#endif
constexpr int kSubPerWG = CMSD_SUB_PER_WG;  // slices per workgroup, all loaded before any is summed
constexpr int kSampleBD = 256;

struct SlicePart {
  double et, ed, q, qd;
};

template <typename T>
__device__ __forceinline__ int64_t unit_first(const Geom& g, int64_t u) {
  return u == 0 ? 0 : (u <= g.nvec ? g.head + (u - 1) * Elem<T>::VEC : g.head + g.nvec * Elem<T>::VEC);
}
template <typename T>
__device__ __forceinline__ int unit_count(const Geom& g, int64_t u) {
  return u == 0 ? g.head : (u <= g.nvec ? Elem<T>::VEC : (u == g.nvec + 1 ? g.tail : 0));
}
// Unit u of the row that defines the units.
template <typename T, bool NT>
__device__ __forceinline__ uint4 unit_raw(const T* row, const Geom& g, int64_t u) {
  using E = Elem<T>;
  if (u >= 1 && u <= g.nvec) {
    const uint4* p = reinterpret_cast<const uint4*>(row + g.head) + (u - 1);
    return NT ? ld_stream(p) : *p;
  }
  const int n = unit_count<T>(g, u);
  return n > 0 ? E::raw_partial(row + unit_first<T>(g, u), n) : E::raw_ninf();
}
// 16 bytes starting `s` bytes into the 32 bytes lo:hi (s in [0, 16), a multiple of
// the element size): whole-word shift by selects, then a byte funnel shift.
__device__ __forceinline__ uint4 window16(const uint4& lo, const uint4& hi, int s) {
  const bool w2 = (s & 8) != 0, w1 = (s & 4) != 0;
  const uint32_t b0 = w2 ? lo.z : lo.x, b1 = w2 ? lo.w : lo.y, b2 = w2 ? hi.x : lo.z, b3 = w2 ? hi.y : lo.w,
                 b4 = w2 ? hi.z : hi.x, b5 = w2 ? hi.w : hi.y;
  const uint32_t c0 = w1 ? b1 : b0, c1 = w1 ? b2 : b1, c2 = w1 ? b3 : b2, c3 = w1 ? b4 : b3, c4 = w1 ? b5 : b4;
  const uint32_t sh = (uint32_t)(s & 3);
  return make_uint4(__builtin_amdgcn_alignbyte(c1, c0, sh), __builtin_amdgcn_alignbyte(c2, c1, sh),
                    __builtin_amdgcn_alignbyte(c3, c2, sh), __builtin_amdgcn_alignbyte(c4, c3, sh));
}

// The same elements of a second row whose 16-byte phase may differ (`same_phase`
// tells whether it matches): one vector load when aligned; otherwise the two
// aligned vectors the 16 bytes straddle (both hold wanted elements), realigned.
template <typename T, bool NT>
__device__ __forceinline__ uint4 unit_raw2(const T* row, const Geom& g, int64_t u, bool same_phase) {
  using E = Elem<T>;
  if (u >= 1 && u <= g.nvec) {
    const T* p = row + g.head + (u - 1) * E::VEC;
    if (same_phase) {
      const uint4* q = reinterpret_cast<const uint4*>(p);
      return NT ? ld_stream(q) : *q;
    }
    const uintptr_t a = reinterpret_cast<uintptr_t>(p);
    const int s = int(a & 15u);
    const uint4* q = reinterpret_cast<const uint4*>(a - (uintptr_t)s);
    const uint4 lo = NT ? ld_stream(q) : q[0];
    const uint4 hi = NT ? ld_stream(q + 1) : q[1];
    return window16(lo, hi, s);
  }
  const int n = unit_count<T>(g, u);
  return n > 0 ? E::raw_partial(row + unit_first<T>(g, u), n) : E::raw_ninf();
}

// What the final-token pass needs of sequence b: the layout check, the accepted
// prefix (first rejection, by ballots over the accept flags), the row(s) of the
// final sample and their normalisers.  Wave 0 reads the sequence's row slots (which
// also carry each drafted position's drafter max and normaliser) in one round trip
// (k_max < 64; longer drafts loop), the result is broadcast through LDS.  nacc = -1
// marks an invalid sequence.
struct SeqInfo {
  int64_t off, tr, dr;
  int nacc, kb;
  float mst, msd, rho0;
  int top1;  // argmax of the final row (GREEDY mode)
};

__device__ __forceinline__ SeqInfo seq_info(const VerifyArgs& a, int b, SeqInfo* lds) {
  const int t = threadIdx.x, lane = t & 63;
  if (t < 64) {
    const int K = a.k_max;
    const int64_t off = a.off[b], off1 = a.off[b + 1];
    const int kb = a.klen[b];
    const RowSlot* S = a.slots + (int64_t)b * (K + 1);
    SeqInfo q{};
    q.nacc = -1;
    const bool ok = kb >= 0 && kb <= K && off >= 0 && off1 == off + kb + 1 && off1 <= a.target_rows;
    // slot j must be this call's row off + j with a consistent flag: 0/1 for drafted
    // positions, -1 for the final row
    auto bad_at = [&](int j, const RowSlot& sl) {
      return j <= kb && (sl.r != (int32_t)(off + j) || (j < kb && sl.acc != 0 && sl.acc != 1) ||
                         (j == kb && sl.acc != -1));
    };
    if (K < 64) {
      const RowSlot sl = lane <= K ? S[lane] : RowSlot{0.f, 1.f, 1, 0, -1, 0.f, 1.f, 0};
      if (ok && __ballot(bad_at(lane, sl)) == 0ull) {
        const unsigned long long rej = __ballot(lane < kb && sl.acc == 0);
        const int j = rej ? __builtin_ctzll(rej) : kb;  // slot of the final row: c, or k_b
        q.nacc = j;
        q.kb = kb;
        q.off = off;
        q.tr = off + j;
        q.dr = (int64_t)b * K + (j < kb ? j : 0);
        q.mst = rl_f(sl.m, j) * kLog2e;
        q.top1 = __builtin_amdgcn_readlane(sl.top1, j);
        if (j < kb) {
          q.msd = rl_f(sl.dm, j) * kLog2e;
          q.rho0 = (float)((double)rl_f(sl.A, j) / (double)rl_f(sl.dA, j));
        }
      }
    } else if (ok) {
      bool bad = false;
      int j = kb;
      for (int base = 0; base <= kb; base += 64) {
        const int jj = base + lane;
        const RowSlot sl = jj <= kb ? S[jj] : RowSlot{0.f, 1.f, 1, 0, -1, 0.f, 1.f, 0};
        if (__ballot(bad_at(jj, sl)) != 0ull) bad = true;
        const unsigned long long rej = __ballot(jj < kb && sl.acc == 0);
        if (rej != 0ull && j == kb) j = base + __builtin_ctzll(rej);
      }
      if (!bad) {
        const RowSlot sl = S[j];
        q.nacc = j;
        q.kb = kb;
        q.off = off;
        q.tr = off + j;
        q.dr = (int64_t)b * K + (j < kb ? j : 0);
        q.mst = sl.m * kLog2e;
        q.top1 = sl.top1;
        if (j < kb) {
          q.msd = sl.dm * kLog2e;
          q.rho0 = (float)((double)sl.A / (double)sl.dA);
        }
      }
    }
    if (lane == 0) *lds = q;
  }
  __syncthreads();
  const SeqInfo r = *lds;
  __syncthreads();
  return r;
}

// seq_info of the single-call pass: wave 0 reads the sequence's row results, drafter
// stats, drafted ids and uniforms (one round trip, k_max < 64) and forms the draft
// length and every accept test (as the separate calls would); with WRITE it also stores
// the draft length and the target-row records.  The slots are only read, so every
// workgroup of the final-token kernels forms the same decisions from them.
template <bool WRITE>
__device__ __forceinline__ SeqInfo seq_info_pass(const VerifyArgs& a, int b, SeqInfo* lds) {
  const int t = threadIdx.x, lane = t & 63;
  if (t < 64) {
    const int K = a.k_max;
    const bool greedy = a.mode == CMSD_MODE_GREEDY;
    const int64_t off = (int64_t)b * (K + 1);
    const PassSlot sl = lane <= K ? a.pslots[off + lane] : PassSlot{1.0, 0.f, -INFINITY, -INFINITY, 0, -1, -1};
    float dmx = 0.f, dA = 1.f, cf = 0.f, u = 0.f;
    int y = -1;
    if (lane < K) {
      const cmsd_row_stats ds = a.dstats[(int64_t)b * K + lane];
      dmx = ds.max_logit;
      dA = ds.sum_exp;
      cf = ds.conf;
      y = a.drafted[(int64_t)b * K + lane];
      if (!greedy) u = a.unif[off + lane];
    }
    // draft length from the confidences, summed in position order in fp64
    double csum = 0.0;
    for (int j = 0; j < K; ++j) csum += (double)rl_f(cf, j);
    const double x = (double)a.alpha * (csum / (double)K) * (double)K;
    const double fl = floor(x);
    const int kb = fl < (double)a.k_min ? a.k_min : (fl > (double)K ? K : (int)fl);
    const int kv = a.adaptive ? kb : K;
    const bool count = a.mode != CMSD_MODE_STANDARD && a.beta > 0;
    int ng = 0, acc = -1;
    if (lane < K && sl.st == 1)
      acc = accept_test(a.mode, a.beta, a.tau_base, a.gamma, count, sl.ngt, sl.gz, sl.zd, sl.m, sl.A, dmx, dA, cf,
                        u, y, sl.top1, &ng);
    const bool bad = __ballot(lane < K && sl.st == -2) != 0ull;
    const unsigned long long rej = __ballot(lane < kv && acc == 0);
    const int c = rej ? __builtin_ctzll(rej) : kv;
    SeqInfo q{};
    q.nacc = bad ? -1 : c;
    q.kb = kv;
    q.off = off;
    q.tr = off + c;
    q.dr = (int64_t)b * K + (c < kv ? c : 0);
    q.mst = rl_f(sl.m, c) * kLog2e;
    q.top1 = __builtin_amdgcn_readlane(sl.top1, c);
    if (c < kv) {
      q.msd = rl_f(dmx, c) * kLog2e;
      q.rho0 = (float)((double)(float)rl_d(sl.A, c) / (double)rl_f(dA, c));  // as from the verify slots
    }
    if (WRITE && lane == 0) a.klen_out[b] = kb;
    if (WRITE && lane <= K) {
      cmsd_target_stats res{};
      res.max_logit = sl.m;
      res.sum_exp = (float)sl.A;
      res.top1 = sl.top1;
      if (sl.st == -2) {
        res = cmsd_target_stats{NAN, NAN, -1, -2, -1, {0, 0, 0}};
      } else if (lane == kv || sl.st == -1) {
        res.n_greater = -1;  // the final row
        res.accept = -1;
      } else {
        res.n_greater = ng;
        res.accept = acc;
      }
      a.tstats[off + lane] = res;
    }
    if (lane == 0) *lds = q;
  }
  __syncthreads();
  const SeqInfo r = *lds;
  __syncthreads();
  return r;
}

// Where the final-token kernels of cmsd_logit_pass find their sequence's decisions:
// in a record that k_pass_decide wrote (large launches), or formed by each of their
// workgroups from the row slots (small launches: one launch fewer).  Verify is the
// separate cmsd_verify, whose decisions come from its own row slots (seq_info).
enum class Src { Verify, Record, Inline };

// The sequence record of the single-call pass sits over the first two row slots of the
// sequence (k_max >= 1), which k_pass_decide has read before it writes the record.
static_assert(sizeof(SeqInfo) <= 2 * sizeof(PassSlot), "a sequence record fits two row slots");
__device__ __forceinline__ SeqInfo* pass_info(const VerifyArgs& a, int b) {
  return reinterpret_cast<SeqInfo*>(a.pslots + (int64_t)b * (a.k_max + 1));
}

// Decisions of the single-call pass, one wave per sequence: draft length, accept
// tests, first rejection (seq_info_pass), the draft length and target-row records;
// the outputs of an invalid sequence and, in GREEDY mode, the final outputs; and the
// sequence record that the final-token kernels read in one load instead of repeating
// the decisions per slice.
__global__ __launch_bounds__(64) void k_pass_decide(VerifyArgs a) {
  __shared__ SeqInfo s_q;
  const int b = blockIdx.x;
  if (b >= a.B) return;
  const SeqInfo q = seq_info_pass<true>(a, b, &s_q);
  if (threadIdx.x == 0) {
    *pass_info(a, b) = q;
    if (q.nacc < 0) {
      a.n_acc[b] = -1;
      a.next_tok[b] = -1;
    } else if (a.mode == CMSD_MODE_GREEDY) {
      a.n_acc[b] = q.nacc;
      a.next_tok[b] = q.top1;
    }
  }
}

// Partial sums of one raw unit: e_t, e_d, q0 and e_d where q0 > 0.
template <typename T, bool RESID>
__device__ __forceinline__ void part_unit(const uint4& rt, const uint4& rd, float mst, float msd, float rho0,
                                          float& at, float& ad, float& aq, float& aqd) {
  using E = Elem<T>;
  constexpr int VEC = E::VEC;
  float ft[VEC], fd[VEC];
  E::unpack(rt, ft);
  if (RESID) E::unpack(rd, fd);
#pragma unroll
  for (int e = 0; e < VEC; ++e) {
    const float et = fexp2(fmaf(ft[e], kLog2e, -mst));
    at += et;
    if (RESID) {
      const float ed = fexp2(fmaf(fd[e], kLog2e, -msd));
      const float q = fmaxf(fmaf(-rho0, ed, et), 0.f);
      ad += ed;
      aq += q;
      aqd += q > 0.f ? ed : 0.f;
    }
  }
}

// NSUB consecutive slices by one wave (lane = its lane index): every unit load of
// every slice is issued before any is summed, so the wave costs one memory latency.
template <typename T, bool RESID, int NSUB>
__device__ __forceinline__ void parts_wave(const T* trow, const T* drow, const Geom& g, bool same_phase,
                                           int64_t u_first, int lane, float mst, float msd, float rho0,
                                           double (&sum)[NSUB][4]) {
  constexpr int UPT = kSliceUnits / 64, NU = NSUB * UPT;
  uint4 rt[NU], rd[NU];
#pragma unroll
  for (int j = 0; j < NU; ++j) {
    const int64_t u = u_first + (int64_t)j * 64 + lane;
    rt[j] = unit_raw<T, true>(trow, g, u);
    if (RESID) rd[j] = unit_raw2<T, true>(drow, g, u, same_phase);
  }
#pragma unroll
  for (int k = 0; k < NSUB; ++k) {
#pragma unroll
    for (int jj = 0; jj < UPT; ++jj) {
      const int j = k * UPT + jj;
      float at = 0.f, ad = 0.f, aq = 0.f, aqd = 0.f;
      part_unit<T, RESID>(rt[j], rd[j], mst, msd, rho0, at, ad, aq, aqd);
      sum[k][0] += (double)at;
      sum[k][1] += (double)ad;
      sum[k][2] += (double)aq;
      sum[k][3] += (double)aqd;
    }
  }
}

template <typename T, Src SRC>
__global__ __launch_bounds__(kPartBD) void k_final_parts(VerifyArgs a, int S, int SW, SlicePart* __restrict__ ws) {
  constexpr int BD = kPartBD;
  __shared__ double sd[kSubPerWG * 4 * (BD / 64)];
  __shared__ SeqInfo s_q;
  const int t = threadIdx.x;
  const int b = blockIdx.x / SW, sl0 = (blockIdx.x % SW) * kSubPerWG;
  if (b >= a.B) return;
  const SeqInfo q = SRC == Src::Record   ? *pass_info(a, b)
                    : SRC == Src::Inline ? seq_info_pass<false>(a, b, &s_q)
                                         : seq_info(a, b, &s_q);
  if (q.nacc < 0) return;
  const bool resid = q.nacc < q.kb;
  const T* trow = reinterpret_cast<const T*>(a.target) + q.tr * a.tstride;
  const T* drow = reinterpret_cast<const T*>(a.draft) + q.dr * a.dstride;
  const bool same_phase = ((reinterpret_cast<uintptr_t>(trow) ^ reinterpret_cast<uintptr_t>(drow)) & 15u) == 0;
  const float mst = q.mst, msd = q.msd, rho0 = q.rho0;
  const Geom g = row_geom(trow, a.V);
  const int64_t nu = g.nvec + 2;
  // wave-level sums per slice (uniform values), one LDS round at the end
  double sum[kSubPerWG][4] = {};
  const int64_t u_first = (int64_t)sl0 * kSliceUnits;
  if (u_first < nu) {
    if (resid)
      parts_wave<T, true, kSubPerWG>(trow, drow, g, same_phase, u_first, t, mst, msd, rho0, sum);
    else
      parts_wave<T, false, kSubPerWG>(trow, trow, g, true, u_first, t, mst, 0.f, 0.f, sum);
  }
  double ws_w[kSubPerWG][4];
#pragma unroll
  for (int k = 0; k < kSubPerWG; ++k)
#pragma unroll
    for (int j = 0; j < 4; ++j) ws_w[k][j] = wave_all_d(sum[k][j], OpSumD());
  constexpr int NW = BD / 64;
  if ((t & 63) == 0) {
#pragma unroll
    for (int k = 0; k < kSubPerWG; ++k)
#pragma unroll
      for (int j = 0; j < 4; ++j) sd[(k * 4 + j) * NW + (t >> 6)] = ws_w[k][j];
  }
  __syncthreads();
  if (t < kSubPerWG * 4) {
    const int k = t >> 2;
    double r = sd[t * NW];
    for (int i = 1; i < NW; ++i) r += sd[t * NW + i];
    if (sl0 + k < S) reinterpret_cast<double*>(ws + (int64_t)b * S + sl0 + k)[t & 3] = r;
  }
}

// Sampling weights of one raw unit: RESID max(0, e_t - rho e_d), else e_t (fp64);
// padding elements weigh exactly 0.
template <typename T, bool RESID>
__device__ __forceinline__ void unit_weights(const uint4& rt, const uint4& rd, float mst, float msd, double rho,
                                             double* q) {
  using E = Elem<T>;
  constexpr int VEC = E::VEC;
  float ft[VEC], fd[VEC];
  E::unpack(rt, ft);
  if (RESID) E::unpack(rd, fd);
#pragma unroll
  for (int e = 0; e < VEC; ++e) {
    const double et = (double)fexp2(fmaf(ft[e], kLog2e, -mst));
    if (RESID) {
      const double ed = (double)fexp2(fmaf(fd[e], kLog2e, -msd));
      const double d = fma(-rho, ed, et);
      q[e] = d > 0.0 ? d : 0.0;
    } else {
      q[e] = et;
    }
  }
}

// Block exclusive scan of one double per thread (wave scan by shuffles, wave totals
// added in order): deterministic.
template <int BD>
__device__ __forceinline__ double block_excl_scan(double v, double* sd) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  double incl = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double up = __shfl_up(incl, o);
    if (lane >= o) incl += up;
  }
  double ex = __shfl_up(incl, 1);
  if (lane == 0) ex = 0.0;
  __syncthreads();
  if (lane == 63) sd[w] = incl;
  __syncthreads();
  double pre = 0.0;
  for (int i = 0; i < w; ++i) pre += sd[i];
  return pre + ex;
}

// Units of one slice per thread of a BD-thread sampling workgroup (one each, and
// none for the threads past the slice, when the workgroup is wider than a slice).
template <int BD>
constexpr int loc_upt() {
  return BD >= kSliceUnits ? 1 : kSliceUnits / BD;
}
static_assert(kSliceUnits % kSampleBD == 0, "a slice splits evenly over the sampling workgroup");

// Smallest element y in units [ulo, uhi) with q_y > 0 and base + C(y) > x, C the
// cumulative weight from ulo in a fixed order: thread t owns the loc_upt<BD>() units
// from ulo + t*loc_upt<BD>() (kept in registers) and sums them unit by unit, a block scan
// orders the threads, and the thread whose span crosses x repeats its own sums
// exactly.  If none qualifies, the last element with q_y > 0.  Returns -1 if every
// weight is 0.  The result passes through *s_y.
template <typename T, bool RESID, int BD>
__device__ __forceinline__ int locate_units(const T* trow, const T* drow, const Geom& g, bool same_phase, int64_t ulo, int64_t uhi,
                            float mst, float msd, double rho, double base, double x, double* sd, int* si,
                            int* s_y) {
  using E = Elem<T>;
  constexpr int VEC = E::VEC, UPT = loc_upt<BD>();
  const int t = threadIdx.x;
  const int64_t u0 = ulo + (int64_t)t * UPT;
  uint4 rt[UPT], rd[UPT];
#pragma unroll
  for (int j = 0; j < UPT; ++j) {
    const bool in = u0 + j < uhi;
    rt[j] = in ? unit_raw<T, false>(trow, g, u0 + j) : E::raw_ninf();
    rd[j] = RESID && in ? unit_raw2<T, false>(drow, g, u0 + j, same_phase) : rt[j];
  }
  double us[UPT];
  double s = 0.0;
#pragma unroll
  for (int j = 0; j < UPT; ++j) {
    double q[VEC];
    unit_weights<T, RESID>(rt[j], rd[j], mst, msd, rho, q);
    double v = 0.0;
#pragma unroll
    for (int e = 0; e < VEC; ++e) v += q[e];
    us[j] = v;
    s += v;
  }
  const double excl = block_excl_scan<BD>(s, sd);
  const double end = base + (excl + s);
  int pick = block_all_i<BD>((s > 0.0 && end > x) ? t : INT32_MAX, OpMinI(), si);
  bool last = false;
  if (pick == INT32_MAX) {
    pick = block_all_i<BD>(s > 0.0 ? t : -1, OpMaxI(), si);
    if (pick < 0) return -1;
    last = true;
  }
  if (t == pick) {
    int y = -1;
    double P = 0.0;
    bool done = false;
#pragma unroll
    for (int j = 0; j < UPT; ++j) {
      const double Pn = P + us[j];
      if (!done && us[j] > 0.0 && (last || base + (excl + Pn) > x)) {
        double q[VEC];
        unit_weights<T, RESID>(rt[j], rd[j], mst, msd, rho, q);
        const int64_t first = unit_first<T>(g, u0 + j);
        double Q = 0.0;
        bool found = false;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          Q += q[e];
          if (!found && q[e] > 0.0 && (last || base + (excl + (P + Q)) > x)) {
            y = int(first + e);
            found = !last;
          }
        }
        done = !last;
      }
      P = Pn;
    }
    *s_y = y;
  }
  __syncthreads();
  const int y = *s_y;
  __syncthreads();
  return y;
}

// Inverse-CDF sample over one row (RESID off) or the residual of a row pair, from
// the row's vocabulary-slice partials P[0..S): rho = sum e_t / sum e_d (fresh sums),
// slice masses corrected to first order in rho - rho0 and scanned in slice order
// (each thread a contiguous run of slices, its first partial kept in registers),
// then an exact scan/locate inside the chosen slice.  A zero residual falls back to
// the target row.  Run by one workgroup of BD threads; s_sc holds 3 doubles, sd
// 2*BD/64 and si BD/64.
template <typename T, int BD>
__device__ __forceinline__ int sample_from_parts(const T* trow, const T* drow, int64_t V, bool resid, float mst, float msd,
                                 float rho0, float u, const SlicePart* __restrict__ P, int S, double* sd, int* si,
                                 double* s_sc, int* s_y, const SlicePart* first = nullptr) {
  const int t = threadIdx.x;
  const bool same_phase = ((reinterpret_cast<uintptr_t>(trow) ^ reinterpret_cast<uintptr_t>(drow)) & 15u) == 0;
  const int slo = (int)((int64_t)t * S / BD), shi = (int)((int64_t)(t + 1) * S / BD);
  // `first`: this thread's first partial, already loaded by the caller
  const SlicePart p0 = first ? *first : (slo < shi ? P[slo] : SlicePart{0.0, 0.0, 0.0, 0.0});
  // fresh normalisers and the exact ratio
  double tot[2] = {0.0, 0.0};
  for (int s = slo; s < shi; ++s) {
    const SlicePart p = s == slo ? p0 : P[s];
    tot[0] += p.et;
    tot[1] += p.ed;
  }
  block_sum_n<BD, 2>(tot, sd);
  const double rho = resid ? tot[0] / tot[1] : 0.0;
  // slice masses (first-order correction of the rho0 sums); a zero residual falls
  // back to the target row itself
  auto mass = [&](int s, bool rs) -> double {
    const SlicePart p = s == slo ? p0 : P[s];
    if (!rs) return p.et;
    const double m = p.q - (rho - (double)rho0) * p.qd;
    return m > 0.0 ? m : 0.0;
  };
  int y = -1;
  const Geom g = row_geom(trow, V);
  const int64_t nu = g.nvec + 2;
  for (int pass = 0; pass < 2 && y < 0; ++pass) {
    double sm = 0.0;
    for (int s = slo; s < shi; ++s) sm += mass(s, resid);
    const double excl = block_excl_scan<BD>(sm, sd);
    const double end = excl + sm;
    const int tlast = block_all_i<BD>(sm > 0.0 ? t : -1, OpMaxI(), si);
    if (tlast < 0) {
      resid = false;  // no residual mass: sample from the target row
      continue;
    }
    if (t == tlast) s_sc[1] = end;
    __syncthreads();
    const double x = (double)u * s_sc[1];
    const int tp = block_all_i<BD>((sm > 0.0 && end > x) ? t : INT32_MAX, OpMinI(), si);
    const int tq = tp == INT32_MAX ? tlast : tp;
    if (t == tq) {
      // the slice inside this thread's run, repeating its sequential sums exactly
      double Pacc = 0.0, sbase = 0.0;
      int sstar = -1;
      for (int s = slo; s < shi; ++s) {
        const double m = mass(s, resid);
        const double Pn = Pacc + m;
        if (m > 0.0) {
          sstar = s;
          sbase = excl + Pacc;
          if (tp != INT32_MAX && excl + Pn > x) break;
        }
        Pacc = Pn;
      }
      s_sc[0] = sbase;
      s_sc[2] = (double)sstar;
    }
    __syncthreads();
    const double sbase = s_sc[0];
    const int64_t ulo = (int64_t)s_sc[2] * kSliceUnits;
    const int64_t uhi = ulo + kSliceUnits < nu ? ulo + kSliceUnits : nu;
    if (resid)
      y = locate_units<T, true, BD>(trow, drow, g, same_phase, ulo, uhi, mst, msd, rho, sbase, x, sd, si, s_y);
    else
      y = locate_units<T, false, BD>(trow, trow, g, true, ulo, uhi, mst, mst, 0.0, sbase, x, sd, si, s_y);
    if (y < 0 && resid) {
      resid = false;
      continue;
    }
    break;
  }
  return y;
}

template <typename T, Src SRC>
__global__ __launch_bounds__(kSampleBD) void k_final_sample(VerifyArgs a, int S, const SlicePart* __restrict__ ws) {
  constexpr int BD = kSampleBD;
  __shared__ double sd[2 * (BD / 64)];
  __shared__ int si[BD / 64];
  __shared__ double s_sc[3];
  __shared__ int s_y;
  __shared__ SeqInfo s_q;
  const int t = threadIdx.x;
  const int b = blockIdx.x;
  if (b >= a.B) return;
  // this thread's first slice partial, written by k_final_parts: its load does not wait
  // for the decisions, so the two round trips overlap (unused for an invalid sequence
  // and in GREEDY mode, where no partials were written; always inside the workspace)
  const int slo = (int)((int64_t)t * S / BD), shi = (int)((int64_t)(t + 1) * S / BD);
  const SlicePart first = slo < shi ? ws[(int64_t)b * S + slo] : SlicePart{0.0, 0.0, 0.0, 0.0};
  const SeqInfo q = SRC == Src::Record   ? *pass_info(a, b)
                    : SRC == Src::Inline ? seq_info_pass<true>(a, b, &s_q)
                                         : seq_info(a, b, &s_q);
  if (SRC == Src::Record && (q.nacc < 0 || a.mode == CMSD_MODE_GREEDY)) return;  // written by k_pass_decide
  if (q.nacc < 0) {
    if (t == 0) {
      a.n_acc[b] = -1;
      a.next_tok[b] = -1;
    }
    return;
  }
  const int nacc = q.nacc;
  if (a.mode == CMSD_MODE_GREEDY) {
    if (t == 0) {
      a.n_acc[b] = nacc;
      a.next_tok[b] = q.top1;
    }
    return;
  }
  const bool resid = nacc < q.kb;
  const T* trow = reinterpret_cast<const T*>(a.target) + q.tr * a.tstride;
  const T* drow = reinterpret_cast<const T*>(a.draft) + q.dr * a.dstride;
  const float u = a.unif[q.off + q.kb];
  const int y = sample_from_parts<T, BD>(trow, drow, a.V, resid, q.mst, q.msd, q.rho0, u, ws + (int64_t)b * S, S, sd,
                                     si, s_sc, &s_y, &first);
  if (t == 0) {
    a.n_acc[b] = nacc;
    a.next_tok[b] = y;
  }
}

// ----------------------------------------------------------------------------- K5 draft sampling
// One exact softmax sample per drafter row (the draws a sampled draft needs):
// vocabulary-slice partials of e = 2^(z log2e - m log2e), then the same slice scan
// and exact in-slice locate as the final token, with u one uniform per row.
// ----------------------------------------------------------------------------- fused pass (small batches)
// The whole dense logit pass in one launch.  The grid is k_row_pass's (drafter rows,
// then target rows, one 256-thread workgroup each).  Every row workgroup publishes its
// record behind a device fence and counts itself into its sequence's counter; the
// workgroup that completes the count (2 k_max + 1 rows) fences again, makes the
// sequence's decisions (seq_info_pass, as k_pass_decide), computes the final row's
// slice partials one wave per slice (parts_wave, as k_final_parts) and samples from
// them (sample_from_parts, as k_final_sample), then sets the counter back to zero.
// The arithmetic is the four-launch pass's, so the outputs are bit-identical to it.
// The fences serialise chip-wide (about 35-50 ns per workgroup), which is why this
// path is for launches of a few hundred rows, where it saves three dependent launches.
constexpr int kFusedBD = 256;
#ifndef CMSD_FUSED_SUB
#define CMSD_FUSED_SUB 2
#endif
constexpr int kFusedSub = CMSD_FUSED_SUB;  // slices per wave and step in the final-token part

template <typename T>
__device__ __forceinline__ void fused_tail(const VerifyArgs& a, int b, int S, SlicePart* __restrict__ ws) {
  constexpr int BD = kFusedBD, NW = BD / 64;
  __shared__ SeqInfo s_q;
  __shared__ double sd[2 * NW];
  __shared__ int si[NW];
  __shared__ double s_sc[3];
  __shared__ int s_y;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const SeqInfo q = seq_info_pass<true>(a, b, &s_q);
  if (q.nacc < 0 || a.mode == CMSD_MODE_GREEDY) {
    if (t == 0) {
      a.n_acc[b] = q.nacc < 0 ? -1 : q.nacc;
      a.next_tok[b] = q.nacc < 0 ? -1 : q.top1;
    }
    return;
  }
  const bool resid = q.nacc < q.kb;
  const T* trow = reinterpret_cast<const T*>(a.target) + q.tr * a.tstride;
  const T* drow = reinterpret_cast<const T*>(a.draft) + q.dr * a.dstride;
  const bool same_phase = ((reinterpret_cast<uintptr_t>(trow) ^ reinterpret_cast<uintptr_t>(drow)) & 15u) == 0;
  const Geom g = row_geom(trow, a.V);
  const int64_t nu = g.nvec + 2;
  SlicePart* P = ws + (int64_t)b * S;
  // kFusedSub consecutive slices per wave and step, all their loads issued first
  for (int sl = w * kFusedSub; sl < S; sl += NW * kFusedSub) {
    double sum[kFusedSub][4] = {};
    const int64_t u_first = (int64_t)sl * kSliceUnits;
    if (u_first < nu) {
      if (resid)
        parts_wave<T, true, kFusedSub>(trow, drow, g, same_phase, u_first, lane, q.mst, q.msd, q.rho0, sum);
      else
        parts_wave<T, false, kFusedSub>(trow, trow, g, true, u_first, lane, q.mst, 0.f, 0.f, sum);
    }
#pragma unroll
    for (int k = 0; k < kFusedSub; ++k) {
      double r[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) r[j] = wave_all_d(sum[k][j], OpSumD());
      if (lane == 0 && sl + k < S) P[sl + k] = SlicePart{r[0], r[1], r[2], r[3]};
    }
  }
  __syncthreads();  // the partials of every slice, written by this workgroup
  const float u = a.unif[q.off + q.kb];
  const int y = sample_from_parts<T, BD>(trow, drow, a.V, resid, q.mst, q.msd, q.rho0, u, P, S, sd, si, s_sc, &s_y);
  if (t == 0) {
    a.n_acc[b] = q.nacc;
    a.next_tok[b] = y;
  }
}

template <typename T>
__global__ __launch_bounds__(kFusedBD) void k_fused_pass(VerifyArgs a, int S, SlicePart* __restrict__ ws,
                                                         int32_t* __restrict__ cnt) {
  __shared__ int s_last;
  const int64_t nd = (int64_t)a.B * a.k_max;
  const int64_t r = blockIdx.x;
  int b;
  if (r < nd) {
    conf_row<T, kFusedBD, false, CMSD_STREAM_DEPTH, kKeepWide<T, CMSD_STREAM_DEPTH>>(
        reinterpret_cast<const T*>(a.draft) + r * a.dstride, a.V, a.ca, a.dstats_out + r, nullptr);
    b = int(r / a.k_max);
  } else {
    target_row<T, kFusedBD, true>(a, r - nd);
    b = int((r - nd) / (a.k_max + 1));
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    __threadfence();  // this row's record is visible before it is counted
    s_last = atomicAdd(cnt + b, 1) == 2 * a.k_max;
  }
  __syncthreads();
  if (!s_last) return;
  __threadfence();  // every other row of the sequence was counted after its record
  if (threadIdx.x == 0) cnt[b] = 0;
  fused_tail<T>(a, b, S, ws);
}

template <typename T>
__global__ __launch_bounds__(kPartBD) void k_draft_parts(const T* __restrict__ logits, int64_t stride, int64_t V,
                                                         const cmsd_row_stats* __restrict__ stats, int S, int SW,
                                                         SlicePart* __restrict__ ws) {
  constexpr int BD = kPartBD;
  __shared__ double sd[kSubPerWG * 4 * (BD / 64)];
  const int t = threadIdx.x;
  const int64_t r = blockIdx.x / SW;
  const int sl0 = (blockIdx.x % SW) * kSubPerWG;
  const T* row = logits + r * stride;
  const Geom g = row_geom(row, V);
  const int64_t nu = g.nvec + 2;
  const float mst = stats[r].max_logit * kLog2e;
  double sum[kSubPerWG][4] = {};
  const int64_t u_first = (int64_t)sl0 * kSliceUnits;
  if (u_first < nu) parts_wave<T, false, kSubPerWG>(row, row, g, true, u_first, threadIdx.x, mst, 0.f, 0.f, sum);
  double w_[kSubPerWG];
#pragma unroll
  for (int k = 0; k < kSubPerWG; ++k) w_[k] = wave_all_d(sum[k][0], OpSumD());
  constexpr int NW = BD / 64;
  if ((t & 63) == 0) {
#pragma unroll
    for (int k = 0; k < kSubPerWG; ++k) sd[k * NW + (t >> 6)] = w_[k];
  }
  __syncthreads();
  if (t < kSubPerWG && sl0 + t < S) {
    double e = sd[t * NW];
    for (int i = 1; i < NW; ++i) e += sd[t * NW + i];
    ws[r * S + sl0 + t] = SlicePart{e, 0.0, 0.0, 0.0};
  }
}

template <typename T>
__global__ __launch_bounds__(kSampleBD) void k_draft_pick(const T* __restrict__ logits, int64_t stride, int64_t V,
                                                          const cmsd_row_stats* __restrict__ stats,
                                                          const float* __restrict__ unif, int S,
                                                          const SlicePart* __restrict__ ws, int32_t* __restrict__ out) {
  constexpr int BD = kSampleBD;
  __shared__ double sd[2 * (BD / 64)];
  __shared__ int si[BD / 64];
  __shared__ double s_sc[3];
  __shared__ int s_y;
  const int64_t r = blockIdx.x;
  const T* row = logits + r * stride;
  const int y = sample_from_parts<T, kSampleBD>(row, row, V, false, stats[r].max_logit * kLog2e, 0.f, 0.f, unif[r], ws + r * S,
                                     S, sd, si, s_sc, &s_y);
  if (threadIdx.x == 0) out[r] = y;
}

// ----------------------------------------------------------------------------- host helpers
bool finite_f(float x) { return x == x && x != INFINITY && x != -INFINITY; }
bool aligned(const void* p, size_t n) { return (reinterpret_cast<uintptr_t>(p) % n) == 0; }
hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }
cmsd_status launched() { return hipGetLastError() == hipSuccess ? CMSD_OK : CMSD_ERR_LAUNCH; }

// Launch-shape overrides of the row kernels, set by cmsd_set_row_shape (0 = chosen
// per launch).  Process-wide; read once per launch.
std::atomic<int> g_row_block{0};
std::atomic<int> g_ring_depth{0};

// Workgroup size of the row kernels (one workgroup per logit row).  A row pays a
// fixed cost (pipeline fill, epilogue reductions, the argmax rescan) besides its
// streaming time, so short rows go to narrower groups, each streaming its row for
// longer, as long as the launch still fills every SIMD with 4 waves; long rows and
// short launches use 256 threads.  cmsd_set_row_shape overrides the choice.
int device_cus() {
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 256;
  if (dev < 64 && cache[dev] > 0) return cache[dev];
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
  if (dev < 64) cache[dev] = n;
  return n;
}
// A launch holds at most 2^32 - 1 work-items (workgroups x threads): the grid size of
// an HSA dispatch is 32-bit.  The entry points reject sizes whose launches would not fit.
bool launch_fits(int64_t groups, int threads) { return groups >= 0 && groups * threads <= (int64_t)UINT32_MAX; }
// A row shape gives way to smaller workgroups on a grid that would not fit otherwise.
int fit_block(int bd, int64_t groups) {
  while (bd > 64 && !launch_fits(groups, bd)) bd >>= 1;
  return bd;
}
int row_block(int64_t n_rows, int64_t row_bytes) {
  if (const int v = g_row_block.load(std::memory_order_relaxed)) return fit_block(v, n_rows);
  const int64_t waves = 16 * (int64_t)device_cus();  // 4 waves on each of 4 SIMDs per CU
  if (row_bytes <= (int64_t)128 << 10) {
    if (n_rows >= waves) return 64;
    if (n_rows >= waves / 2) return 128;
  }
  return fit_block(256, n_rows);
}

// Rounds in flight per thread for a streaming-row launch.  Long launches (several
// generations of workgroups: at least 16 rows per compute unit for the joint row pass,
// 32 for the confidence pass alone, as 8448 rows of 128256 logits in one pass or 8192
// drafter rows of 32000) stream better with three rounds in flight; shorter ones keep
// two, whose smaller register count lets more of their rows run at once.  The depth only schedules loads: the
// arithmetic, and so every result, is the same.  cmsd_set_row_shape forces it.
#ifndef CMSD_DEEP_DEPTH
#define CMSD_DEEP_DEPTH 3
#endif
bool deep_ring(int64_t n_rows, int rows_per_cu) {
  if (const int d = g_ring_depth.load(std::memory_order_relaxed)) return d == 3;
  return n_rows >= rows_per_cu * (int64_t)device_cus();
}

// Workgroups per confidence launch: the launch's work-items (workgroups x threads) stay
// below 2^32, and the kernel's loop over rows takes any rows beyond.  (Below the cap
// the loop runs once; a kernel of one row per workgroup and no loop gets more waves
// per SIMD from fewer registers and measured slower on 8192 rows of 32000 logits.)
constexpr int64_t kConfMaxGrid = (int64_t)1 << 22;

template <typename T, bool VAR, int DEPTH>
void launch_confidence_d(int bd, const T* logits, int64_t n_rows, int64_t V, int64_t stride, const ConfArgs& a,
                         cmsd_row_stats* out, float* var, hipStream_t st) {
  const dim3 grid((unsigned)(n_rows < kConfMaxGrid ? n_rows : kConfMaxGrid));
  if (bd == 64)
    hipLaunchKernelGGL((k_confidence<T, 64, VAR, DEPTH>), grid, dim3(64), 0, st, logits, n_rows, V, stride, a, out,
                       var);
  else if (bd == 128)
    hipLaunchKernelGGL((k_confidence<T, 128, VAR, DEPTH>), grid, dim3(128), 0, st, logits, n_rows, V, stride, a, out,
                       var);
  else
    hipLaunchKernelGGL((k_confidence<T, 256, VAR, DEPTH>), grid, dim3(256), 0, st, logits, n_rows, V, stride, a, out,
                       var);
}
template <typename T, bool VAR>
void launch_confidence(int bd, const T* logits, int64_t n_rows, int64_t V, int64_t stride, const ConfArgs& a,
                       cmsd_row_stats* out, float* var, hipStream_t st) {
  if (deep_ring(n_rows, 32))
    launch_confidence_d<T, VAR, CMSD_DEEP_DEPTH>(bd, logits, n_rows, V, stride, a, out, var, st);
  else
    launch_confidence_d<T, VAR, CMSD_STREAM_DEPTH>(bd, logits, n_rows, V, stride, a, out, var, st);
}

template <typename T, int DEPTH>
void launch_target_rows_d(int bd, const VerifyArgs& a, hipStream_t st) {
  const dim3 grid((unsigned)((int64_t)a.B * (a.k_max + 1)));  // one workgroup per (sequence, position)
  if (bd == 64)
    hipLaunchKernelGGL((k_target_rows<T, 64, DEPTH>), grid, dim3(64), 0, st, a);
  else if (bd == 128)
    hipLaunchKernelGGL((k_target_rows<T, 128, DEPTH>), grid, dim3(128), 0, st, a);
  else
    hipLaunchKernelGGL((k_target_rows<T, 256, DEPTH>), grid, dim3(256), 0, st, a);
}
// The packed target rows of cmsd_verify: two rounds in flight (three measured slower
// on 3097 rows of 32000 bf16 logits), three only when forced.
template <typename T>
void launch_target_rows(int bd, const VerifyArgs& a, hipStream_t st) {
  if (g_ring_depth.load(std::memory_order_relaxed) == 3)
    launch_target_rows_d<T, CMSD_DEEP_DEPTH>(bd, a, st);
  else
    launch_target_rows_d<T, CMSD_STREAM_DEPTH>(bd, a, st);
}

// The joint row pass.  With events, they are recorded on the stream just before and
// just after the launch, so the caller can time the launch alone.  A failed record
// stays the thread's last HIP error, which the call's launched() reports.
template <typename K>
void launch_rows(K kernel, int64_t rows, int bd, const VerifyArgs& a, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
  const dim3 grid((unsigned)rows), block((unsigned)bd);
  if (e0) (void)hipEventRecord(e0, st);
  hipLaunchKernelGGL(kernel, grid, block, 0, st, a);
  if (e0) (void)hipEventRecord(e1, st);
}
template <typename T, int DEPTH>
void launch_row_pass_d(int bd, const VerifyArgs& a, int64_t rows, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
  if (bd == 64)
    launch_rows(k_row_pass<T, 64, DEPTH>, rows, bd, a, st, e0, e1);
  else if (bd == 128)
    launch_rows(k_row_pass<T, 128, DEPTH>, rows, bd, a, st, e0, e1);
  else
    launch_rows(k_row_pass<T, 256, DEPTH>, rows, bd, a, st, e0, e1);
}
template <typename T>
void launch_row_pass(int bd, const VerifyArgs& a, int64_t rows, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
  if (deep_ring(rows, 16))
    launch_row_pass_d<T, CMSD_DEEP_DEPTH>(bd, a, rows, st, e0, e1);
  else
    launch_row_pass_d<T, CMSD_STREAM_DEPTH>(bd, a, rows, st, e0, e1);
}

// Number of vocabulary slices of the final-token pass: units are 16-byte vectors
// plus a head and a tail unit (the head shortens the vector run, so nvec + 2 is at
// most vocab / VEC + 2).  The workspace is sized for fp32, the dtype with most units.
int verify_slices(int64_t vocab, int elem_bytes) {
  const int64_t units = vocab / (16 / elem_bytes) + 2;
  return (int)((units + kSliceUnits - 1) / kSliceUnits);
}

// Checked confidence parameters: each lambda in [0,1] with |sum - 1| <= 1e-6 and a
// finite beta_margin > 0.
bool conf_args(const cmsd_conf_params* p, int64_t vocab, ConfArgs& a) {
  const float l1 = p->lambda_ent, l2 = p->lambda_margin, l3 = p->lambda_soft;
  if (!(l1 >= 0.f && l1 <= 1.f && l2 >= 0.f && l2 <= 1.f && l3 >= 0.f && l3 <= 1.f)) return false;
  if (fabs((double)l1 + (double)l2 + (double)l3 - 1.0) > 1e-6) return false;
  if (!finite_f(p->beta_margin) || !(p->beta_margin > 0.f)) return false;
  a = ConfArgs{l1, l2, l3, p->beta_margin, 1.0 / log((double)vocab), 1.0 / (1.0 - 1.0 / (double)vocab)};
  return true;
}
bool draft_params_ok(const cmsd_draft_params* p) {
  return p->k_min >= 1 && p->k_min <= p->k_max && p->k_max <= 4096 && finite_f(p->alpha) && p->alpha > 0.f &&
         p->alpha <= 1.f;
}
bool verify_params_ok(const cmsd_verify_params* p) {
  return (p->mode == CMSD_MODE_STANDARD || p->mode == CMSD_MODE_CM || p->mode == CMSD_MODE_GREEDY) &&
         p->top_beta >= 0 && finite_f(p->tau_base) && finite_f(p->gamma);
}

cmsd_status confidence_impl(const void* logits, int32_t dtype, int64_t n_rows, int64_t vocab, int64_t row_stride,
                            const cmsd_conf_params* params, cmsd_row_stats* stats, float* logit_var, bool want_var,
                            void* stream) {
  if (dtype != CMSD_F32 && dtype != CMSD_BF16) return CMSD_ERR_DTYPE;
  if (!params) return CMSD_ERR_ARG;
  if (n_rows < 0 || n_rows > INT32_MAX || vocab < 2 || vocab > INT32_MAX || row_stride < vocab) return CMSD_ERR_ARG;
  ConfArgs a;
  if (!conf_args(params, vocab, a)) return CMSD_ERR_ARG;
  const size_t es = dtype == CMSD_F32 ? 4 : 2;
  if (n_rows == 0) return CMSD_OK;
  if (!logits || !stats || !aligned(logits, es) || !aligned(stats, 4)) return CMSD_ERR_ARG;
  if (want_var && (!logit_var || !aligned(logit_var, 4))) return CMSD_ERR_ARG;
  if (row_stride > INT64_MAX / n_rows) return CMSD_ERR_ARG;
  const int bd = row_block(n_rows, vocab * (int64_t)es);
  const hipStream_t st = as_stream(stream);
  if (dtype == CMSD_F32) {
    const float* p = static_cast<const float*>(logits);
    if (want_var) launch_confidence<float, true>(bd, p, n_rows, vocab, row_stride, a, stats, logit_var, st);
    else launch_confidence<float, false>(bd, p, n_rows, vocab, row_stride, a, stats, nullptr, st);
  } else {
    const Bf16* p = static_cast<const Bf16*>(logits);
    if (want_var) launch_confidence<Bf16, true>(bd, p, n_rows, vocab, row_stride, a, stats, logit_var, st);
    else launch_confidence<Bf16, false>(bd, p, n_rows, vocab, row_stride, a, stats, nullptr, st);
  }
  return launched();
}

// Checks the arguments of the single-call pass (all but its workspace) and fills its
// kernel arguments; bind_pass_workspace completes them.
cmsd_status pass_setup(const void* draft_logits, int64_t draft_stride, const void* target_logits,
                       int64_t target_stride, const int32_t* drafted, const float* uniforms, int32_t dtype,
                       int32_t batch, int32_t k_max, int64_t vocab, const cmsd_conf_params* conf,
                       const cmsd_draft_params* draft, const cmsd_verify_params* verify, int32_t adaptive,
                       cmsd_row_stats* draft_stats, int32_t* draft_len, cmsd_target_stats* target_stats,
                       int32_t* n_accepted, int32_t* next_token, VerifyArgs& a) {
  if (dtype != CMSD_F32 && dtype != CMSD_BF16) return CMSD_ERR_DTYPE;
  if (!conf || !draft || !verify) return CMSD_ERR_ARG;
  if (batch < 0 || k_max < 1 || k_max > 63 || vocab < 2 || vocab > INT32_MAX) return CMSD_ERR_ARG;
  if (adaptive != 0 && adaptive != 1) return CMSD_ERR_ARG;
  if (!conf_args(conf, vocab, a.ca) || !draft_params_ok(draft) || draft->k_max != k_max || !verify_params_ok(verify))
    return CMSD_ERR_ARG;
  if (draft_stride < vocab || target_stride < vocab) return CMSD_ERR_ARG;
  if (batch == 0) return CMSD_OK;
  const size_t es = dtype == CMSD_F32 ? 4 : 2;
  const int64_t drows = (int64_t)batch * k_max, trows = (int64_t)batch * (k_max + 1);
  if (!launch_fits(drows + trows, 64) || draft_stride > INT64_MAX / drows || target_stride > INT64_MAX / trows)
    return CMSD_ERR_ARG;
  if (!launch_fits((int64_t)batch * verify_slices(vocab, 4), kPartBD) || !launch_fits(batch, kSampleBD))
    return CMSD_ERR_ARG;
  if (!draft_logits || !target_logits || !drafted || (!uniforms && verify->mode != CMSD_MODE_GREEDY) ||
      !draft_stats || !draft_len || !target_stats || !n_accepted || !next_token)
    return CMSD_ERR_ARG;
  if (!aligned(draft_logits, es) || !aligned(target_logits, es) || !aligned(drafted, 4) || !aligned(uniforms, 4) ||
      !aligned(draft_stats, 4) || !aligned(draft_len, 4) || !aligned(target_stats, 4) || !aligned(n_accepted, 4) ||
      !aligned(next_token, 4))
    return CMSD_ERR_ARG;
  a.draft = draft_logits;
  a.dstride = draft_stride;
  a.dstats = draft_stats;
  a.dstats_out = draft_stats;
  a.target = target_logits;
  a.tstride = target_stride;
  a.target_rows = trows;
  a.drafted = drafted;
  a.unif = uniforms;
  a.B = batch;
  a.k_max = k_max;
  a.V = vocab;
  a.mode = verify->mode;
  a.beta = verify->top_beta;
  a.tau_base = verify->tau_base;
  a.gamma = verify->gamma;
  a.tstats = target_stats;
  a.n_acc = n_accepted;
  a.next_tok = next_token;
  a.klen_out = draft_len;
  a.k_min = draft->k_min;
  a.alpha = draft->alpha;
  a.adaptive = adaptive;
  return CMSD_OK;
}

// The caller's workspace of the single-call pass: per sequence, slice records first
// (sized for fp32, the dtype with most slices), then the row slots.
cmsd_status bind_pass_workspace(VerifyArgs& a, void* workspace, size_t workspace_bytes, size_t workspace_need) {
  if (!workspace || workspace_need == 0 || workspace_bytes < workspace_need || !aligned(workspace, 8))
    return CMSD_ERR_ARG;
  static_assert(sizeof(PassSlot) == sizeof(RowSlot), "the pass uses the verify workspace layout");
  a.pslots = reinterpret_cast<PassSlot*>(static_cast<SlicePart*>(workspace) + (size_t)a.B * verify_slices(a.V, 4));
  return CMSD_OK;
}

// The final-token pair of cmsd_logit_pass, its decisions found as SRC says.
template <typename T, Src SRC>
void launch_final(const VerifyArgs& a, int S, int SW, SlicePart* ws, hipStream_t st) {
  const unsigned gp = (unsigned)((int64_t)a.B * SW);
  hipLaunchKernelGGL((k_final_parts<T, SRC>), dim3(gp), dim3(kPartBD), 0, st, a, S, SW, ws);
  hipLaunchKernelGGL((k_final_sample<T, SRC>), dim3((unsigned)a.B), dim3(kSampleBD), 0, st, a, S, ws);
}

// Whether the final-token workgroups of cmsd_logit_pass form their sequence's decisions
// themselves instead of reading k_pass_decide's record: up to 32 slice waves per compute
// unit the launch saved outweighs the repeated decisions (8 or 64 sequences of 8 drafts
// at V = 32000 to 152064); 256 sequences at V = 128256 (63 slices each: 63 waves per
// unit) keep the decision kernel.
// cmsd_set_pass_decisions forces either (0 = chosen per call, 1 = record, 2 = inline).
std::atomic<int> g_pass_decisions{0};

// Timing events armed by cmsd_set_row_events for the next cmsd_logit_pass call of this
// host thread (a measurement hook kept out of the call's own arguments).
thread_local hipEvent_t t_row_events[2] = {nullptr, nullptr};
bool inline_decisions(unsigned slice_waves) {
  if (const int m = g_pass_decisions.load(std::memory_order_relaxed)) return m == 2;
  return slice_waves <= 32u * (unsigned)device_cus();
}

// The launches of cmsd_logit_pass on a bound workspace: the joint row pass (bracketed
// by the caller's events, if any), then either the final-token pair forming the
// decisions in its workgroups (small launches), or the per-sequence decisions followed
// by the final-token pair (not in GREEDY mode, whose final token is the row's top token).
cmsd_status enqueue_logit_pass(const VerifyArgs& a, int32_t dtype, void* workspace, hipEvent_t e0, hipEvent_t e1,
                               hipStream_t st) {
  const int es = dtype == CMSD_F32 ? 4 : 2;
  const int64_t drows = (int64_t)a.B * a.k_max, trows = (int64_t)a.B * (a.k_max + 1);
  const int S = verify_slices(a.V, es);
  const int SW = (S + kSubPerWG - 1) / kSubPerWG;
  SlicePart* ws = static_cast<SlicePart*>(workspace);
  const unsigned gp = (unsigned)((int64_t)a.B * SW);
  const int bd = row_block(drows + trows, a.V * (int64_t)es);
  if (dtype == CMSD_F32)
    launch_row_pass<float>(bd, a, drows + trows, st, e0, e1);
  else
    launch_row_pass<Bf16>(bd, a, drows + trows, st, e0, e1);
  if (a.mode != CMSD_MODE_GREEDY && inline_decisions(gp)) {
    if (dtype == CMSD_F32)
      launch_final<float, Src::Inline>(a, S, SW, ws, st);
    else
      launch_final<Bf16, Src::Inline>(a, S, SW, ws, st);
    return launched();
  }
  hipLaunchKernelGGL(k_pass_decide, dim3((unsigned)a.B), dim3(64), 0, st, a);
  if (a.mode == CMSD_MODE_GREEDY) return launched();
  if (dtype == CMSD_F32)
    launch_final<float, Src::Record>(a, S, SW, ws, st);
  else
    launch_final<Bf16, Src::Record>(a, S, SW, ws, st);
  return launched();
}

// ----------------------------------------------------------------------------- static scratch
// The workspace of cmsd_logit_pass_noalloc: one array per device, held from the
// library's first use on that device until the process ends.  Host code never passes
// the array's name to a kernel (on the host it names a stand-in, not device memory):
// its device address is looked up once per device with hipGetSymbolAddress, with that
// device current, and kept.  Every no-allocation call on a device shares its array.
static __device__ __align__(256) unsigned char scratch[CMSD_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

// Device address of the current device's scratch array; nullptr on a HIP error.
void* scratch_ptr() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  void* p = g_scratch[dev].load(std::memory_order_acquire);
  if (p) return p;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  p = g_scratch[dev].load(std::memory_order_relaxed);
  if (!p) {
    void* q = nullptr;
    if (hipGetSymbolAddress(&q, HIP_SYMBOL(scratch)) != hipSuccess || !q) {
      (void)hipGetLastError();
      return nullptr;
    }
    p = q;
    g_scratch[dev].store(p, std::memory_order_release);
  }
  return p;
}

}  // namespace

// ----------------------------------------------------------------------------- C ABI
extern "C" {

const char* cmsd_status_string(cmsd_status s) {
  switch (s) {
    case CMSD_OK: return "ok";
    case CMSD_ERR_ARG: return "invalid argument";
    case CMSD_ERR_DTYPE: return "unknown logit dtype";
    case CMSD_ERR_LAUNCH: return "kernel launch failed";
    case CMSD_ERR_SIZE: return "problem larger than the static scratch";
  }
  return "unknown status";
}

int32_t cmsd_version(void) { return (1 << 16) | 7; }

size_t cmsd_draft_sample_workspace_bytes(int64_t n_rows, int64_t vocab) {
  if (n_rows <= 0 || n_rows > INT32_MAX || vocab < 2 || vocab > INT32_MAX) return 0;
  return (size_t)n_rows * (size_t)verify_slices(vocab, 4) * sizeof(SlicePart);
}

cmsd_status cmsd_draft_sample(const void* logits, int32_t dtype, int64_t n_rows, int64_t vocab, int64_t row_stride,
                              const cmsd_row_stats* stats, const float* uniforms, int32_t* drafted, void* workspace,
                              size_t workspace_bytes, void* stream) {
  if (dtype != CMSD_F32 && dtype != CMSD_BF16) return CMSD_ERR_DTYPE;
  if (n_rows < 0 || n_rows > INT32_MAX || vocab < 2 || vocab > INT32_MAX || row_stride < vocab) return CMSD_ERR_ARG;
  if (n_rows == 0) return CMSD_OK;
  const size_t es = dtype == CMSD_F32 ? 4 : 2;
  if (!logits || !stats || !uniforms || !drafted || !workspace) return CMSD_ERR_ARG;
  if (!aligned(logits, es) || !aligned(stats, 4) || !aligned(uniforms, 4) || !aligned(drafted, 4) ||
      !aligned(workspace, 8))
    return CMSD_ERR_ARG;
  if (workspace_bytes < cmsd_draft_sample_workspace_bytes(n_rows, vocab)) return CMSD_ERR_ARG;
  if (row_stride > INT64_MAX / n_rows) return CMSD_ERR_ARG;
  const int S = verify_slices(vocab, (int)es);
  const int SW = (S + kSubPerWG - 1) / kSubPerWG;
  if (!launch_fits(n_rows * SW, kPartBD) || !launch_fits(n_rows, kSampleBD)) return CMSD_ERR_ARG;
  SlicePart* ws = static_cast<SlicePart*>(workspace);
  const hipStream_t st = as_stream(stream);
  const dim3 gp((unsigned)(n_rows * SW)), gr((unsigned)n_rows);
  if (dtype == CMSD_F32) {
    hipLaunchKernelGGL((k_draft_parts<float>), gp, dim3(kPartBD), 0, st, static_cast<const float*>(logits), row_stride,
                       vocab, stats, S, SW, ws);
    hipLaunchKernelGGL((k_draft_pick<float>), gr, dim3(kSampleBD), 0, st, static_cast<const float*>(logits),
                       row_stride, vocab, stats, uniforms, S, ws, drafted);
  } else {
    hipLaunchKernelGGL((k_draft_parts<Bf16>), gp, dim3(kPartBD), 0, st, static_cast<const Bf16*>(logits), row_stride,
                       vocab, stats, S, SW, ws);
    hipLaunchKernelGGL((k_draft_pick<Bf16>), gr, dim3(kSampleBD), 0, st, static_cast<const Bf16*>(logits),
                       row_stride, vocab, stats, uniforms, S, ws, drafted);
  }
  return launched();
}

size_t cmsd_verify_workspace_bytes(int32_t batch, int32_t k_max, int64_t vocab) {
  static_assert(sizeof(RowSlot) == 32 && sizeof(SlicePart) == 32, "workspace record sizes");
  if (batch <= 0 || k_max < 1 || k_max > 4096 || vocab < 2 || vocab > INT32_MAX) return 0;
  return (size_t)batch * ((size_t)verify_slices(vocab, 4) * sizeof(SlicePart) + (size_t)(k_max + 1) * sizeof(RowSlot));
}

cmsd_status cmsd_confidence(const void* logits, int32_t dtype, int64_t n_rows, int64_t vocab, int64_t row_stride,
                            const cmsd_conf_params* params, cmsd_row_stats* stats, void* stream) {
  return confidence_impl(logits, dtype, n_rows, vocab, row_stride, params, stats, nullptr, false, stream);
}

cmsd_status cmsd_confidence_var(const void* logits, int32_t dtype, int64_t n_rows, int64_t vocab,
                                int64_t row_stride, const cmsd_conf_params* params, cmsd_row_stats* stats,
                                float* logit_var, void* stream) {
  return confidence_impl(logits, dtype, n_rows, vocab, row_stride, params, stats, logit_var, true, stream);
}

cmsd_status cmsd_draft_len(const cmsd_row_stats* stats, int32_t batch, const cmsd_draft_params* params,
                           int32_t* draft_len, int32_t* target_offsets, void* stream) {
  if (!params || batch < 0 || !draft_params_ok(params)) return CMSD_ERR_ARG;
  const int k_min = params->k_min, k_max = params->k_max;
  if ((int64_t)batch * (k_max + 1) > INT32_MAX) return CMSD_ERR_ARG;
  if (!target_offsets || !aligned(target_offsets, 4)) return CMSD_ERR_ARG;
  if (batch > 0 && (!stats || !draft_len || !aligned(stats, 4) || !aligned(draft_len, 4))) return CMSD_ERR_ARG;
  hipLaunchKernelGGL(k_draft_len, dim3(1), dim3(kDraftBD), 0, as_stream(stream), stats, batch, k_min, k_max,
                     params->alpha, draft_len, target_offsets);
  return launched();
}

cmsd_status cmsd_verify(const void* draft_logits, int64_t draft_stride, const cmsd_row_stats* draft_stats,
                        const void* target_logits, int64_t target_stride, int64_t target_rows,
                        const int32_t* target_offsets, const int32_t* draft_len, const int32_t* drafted,
                        const float* uniforms, int32_t dtype, int32_t batch, int32_t k_max, int64_t vocab,
                        const cmsd_verify_params* params, cmsd_target_stats* target_stats, int32_t* n_accepted,
                        int32_t* next_token, void* workspace, size_t workspace_bytes, void* stream) {
  if (dtype != CMSD_F32 && dtype != CMSD_BF16) return CMSD_ERR_DTYPE;
  if (!params) return CMSD_ERR_ARG;
  if (batch < 0 || k_max < 1 || k_max > 4096 || vocab < 2 || vocab > INT32_MAX) return CMSD_ERR_ARG;
  if (!verify_params_ok(params)) return CMSD_ERR_ARG;
  if (batch == 0) return CMSD_OK;
  if (target_rows < 1 || target_rows > INT32_MAX) return CMSD_ERR_ARG;
  if (draft_stride < vocab || target_stride < vocab) return CMSD_ERR_ARG;
  if (!launch_fits((int64_t)batch * (k_max + 1), 64) || !launch_fits(batch, kSampleBD)) return CMSD_ERR_ARG;
  const size_t es = dtype == CMSD_F32 ? 4 : 2;
  if (!draft_logits || !draft_stats || !target_logits || !target_offsets || !draft_len || !drafted ||
      (!uniforms && params->mode != CMSD_MODE_GREEDY) ||
      !target_stats || !n_accepted || !next_token || !workspace)
    return CMSD_ERR_ARG;
  if (workspace_bytes < cmsd_verify_workspace_bytes(batch, k_max, vocab) || !aligned(workspace, 8)) return CMSD_ERR_ARG;
  if (!launch_fits((int64_t)batch * verify_slices(vocab, 4), kPartBD)) return CMSD_ERR_ARG;
  if (!aligned(draft_logits, es) || !aligned(target_logits, es) || !aligned(draft_stats, 4) ||
      !aligned(target_offsets, 4) || !aligned(draft_len, 4) || !aligned(drafted, 4) || !aligned(uniforms, 4) ||
      !aligned(target_stats, 4) || !aligned(n_accepted, 4) || !aligned(next_token, 4))
    return CMSD_ERR_ARG;
  VerifyArgs a;
  a.draft = draft_logits;
  a.dstride = draft_stride;
  a.dstats = draft_stats;
  a.target = target_logits;
  a.tstride = target_stride;
  a.target_rows = target_rows;
  a.off = target_offsets;
  a.klen = draft_len;
  a.drafted = drafted;
  a.unif = uniforms;
  a.B = batch;
  a.k_max = k_max;
  a.V = vocab;
  a.mode = params->mode;
  a.beta = params->top_beta;
  a.tau_base = params->tau_base;
  a.gamma = params->gamma;
  a.tstats = target_stats;
  a.n_acc = n_accepted;
  a.next_tok = next_token;
  const hipStream_t st = as_stream(stream);
  const int S = verify_slices(vocab, (int)es);
  const int SW = (S + kSubPerWG - 1) / kSubPerWG;
  SlicePart* ws = static_cast<SlicePart*>(workspace);
  a.slots = reinterpret_cast<RowSlot*>(ws + (size_t)batch * verify_slices(vocab, 4));
  const unsigned gp = (unsigned)((int64_t)batch * SW);
  // the shape suits the scored rows; the grid covers every (sequence, position)
  const int bd = fit_block(row_block(target_rows, vocab * (int64_t)es), (int64_t)batch * (k_max + 1));
  if (dtype == CMSD_F32) {
    launch_target_rows<float>(bd, a, st);
    if (a.mode != CMSD_MODE_GREEDY)
      hipLaunchKernelGGL((k_final_parts<float, Src::Verify>), dim3(gp), dim3(kPartBD), 0, st, a, S, SW, ws);
    hipLaunchKernelGGL((k_final_sample<float, Src::Verify>), dim3((unsigned)batch), dim3(kSampleBD), 0, st, a, S, ws);
  } else {
    launch_target_rows<Bf16>(bd, a, st);
    if (a.mode != CMSD_MODE_GREEDY)
      hipLaunchKernelGGL((k_final_parts<Bf16, Src::Verify>), dim3(gp), dim3(kPartBD), 0, st, a, S, SW, ws);
    hipLaunchKernelGGL((k_final_sample<Bf16, Src::Verify>), dim3((unsigned)batch), dim3(kSampleBD), 0, st, a, S, ws);
  }
  return launched();
}

cmsd_status cmsd_logit_pass(const void* draft_logits, int64_t draft_stride, const void* target_logits,
                            int64_t target_stride, const int32_t* drafted, const float* uniforms, int32_t dtype,
                            int32_t batch, int32_t k_max, int64_t vocab, const cmsd_conf_params* conf,
                            const cmsd_draft_params* draft, const cmsd_verify_params* verify, int32_t adaptive,
                            cmsd_row_stats* draft_stats, int32_t* draft_len, cmsd_target_stats* target_stats,
                            int32_t* n_accepted, int32_t* next_token, void* workspace, size_t workspace_bytes,
                            void* stream) {
  // the events armed by cmsd_set_row_events serve this call only, whatever its outcome
  const hipEvent_t e0 = t_row_events[0], e1 = t_row_events[1];
  t_row_events[0] = t_row_events[1] = nullptr;
  VerifyArgs a{};
  cmsd_status e = pass_setup(draft_logits, draft_stride, target_logits, target_stride, drafted, uniforms, dtype,
                             batch, k_max, vocab, conf, draft, verify, adaptive, draft_stats, draft_len, target_stats,
                             n_accepted, next_token, a);
  if (e != CMSD_OK || batch == 0) return e;
  e = bind_pass_workspace(a, workspace, workspace_bytes, cmsd_verify_workspace_bytes(batch, k_max, vocab));
  if (e != CMSD_OK) return e;
  return enqueue_logit_pass(a, dtype, workspace, e0, e1, as_stream(stream));
}

cmsd_status cmsd_set_row_events(void* const* row_events) {
  if (row_events && (!row_events[0] || !row_events[1])) return CMSD_ERR_ARG;
  t_row_events[0] = row_events ? static_cast<hipEvent_t>(row_events[0]) : nullptr;
  t_row_events[1] = row_events ? static_cast<hipEvent_t>(row_events[1]) : nullptr;
  return CMSD_OK;
}

cmsd_status cmsd_logit_pass_noalloc(const void* draft_logits, int64_t draft_stride, const void* target_logits,
                                    int64_t target_stride, const int32_t* drafted, const float* uniforms,
                                    int32_t dtype, int32_t batch, int32_t k_max, int64_t vocab,
                                    const cmsd_conf_params* conf, const cmsd_draft_params* draft,
                                    const cmsd_verify_params* verify, int32_t adaptive, cmsd_row_stats* draft_stats,
                                    int32_t* draft_len, cmsd_target_stats* target_stats, int32_t* n_accepted,
                                    int32_t* next_token, void* stream) {
  VerifyArgs a{};
  cmsd_status e = pass_setup(draft_logits, draft_stride, target_logits, target_stride, drafted, uniforms, dtype,
                             batch, k_max, vocab, conf, draft, verify, adaptive, draft_stats, draft_len, target_stats,
                             n_accepted, next_token, a);
  if (e != CMSD_OK || batch == 0) return e;
  const size_t need = cmsd_verify_workspace_bytes(batch, k_max, vocab);
  if (need > (size_t)CMSD_STATIC_SCRATCH_BYTES) return CMSD_ERR_SIZE;
  void* ws = scratch_ptr();
  if (!ws) return CMSD_ERR_LAUNCH;
  e = bind_pass_workspace(a, ws, (size_t)CMSD_STATIC_SCRATCH_BYTES, need);
  if (e != CMSD_OK) return e;
  return enqueue_logit_pass(a, dtype, ws, nullptr, nullptr, as_stream(stream));
}

cmsd_status cmsd_set_pass_decisions(int32_t mode) {
  if (mode < 0 || mode > 2) return CMSD_ERR_ARG;
  g_pass_decisions.store(mode, std::memory_order_relaxed);
  return CMSD_OK;
}

cmsd_status cmsd_set_row_shape(int32_t threads, int32_t ring_depth) {
  if (threads != 0 && threads != 64 && threads != 128 && threads != 256) return CMSD_ERR_ARG;
  if (ring_depth != 0 && ring_depth != 2 && ring_depth != 3) return CMSD_ERR_ARG;
  g_row_block.store(threads, std::memory_order_relaxed);
  g_ring_depth.store(ring_depth, std::memory_order_relaxed);
  return CMSD_OK;
}

size_t cmsd_logit_pass_fused_workspace_bytes(int32_t batch, int32_t k_max, int64_t vocab) {
  const size_t v = cmsd_verify_workspace_bytes(batch, k_max, vocab);
  if (v == 0 || k_max > 63) return 0;
  return v + (((size_t)batch * sizeof(int32_t) + 7u) & ~(size_t)7u);
}

cmsd_status cmsd_logit_pass_fused(const void* draft_logits, int64_t draft_stride, const void* target_logits,
                                  int64_t target_stride, const int32_t* drafted, const float* uniforms,
                                  int32_t dtype, int32_t batch, int32_t k_max, int64_t vocab,
                                  const cmsd_conf_params* conf, const cmsd_draft_params* draft,
                                  const cmsd_verify_params* verify, int32_t adaptive, cmsd_row_stats* draft_stats,
                                  int32_t* draft_len, cmsd_target_stats* target_stats, int32_t* n_accepted,
                                  int32_t* next_token, void* workspace, size_t workspace_bytes, void* stream) {
  VerifyArgs a{};
  cmsd_status e = pass_setup(draft_logits, draft_stride, target_logits, target_stride, drafted, uniforms, dtype,
                             batch, k_max, vocab, conf, draft, verify, adaptive, draft_stats, draft_len, target_stats,
                             n_accepted, next_token, a);
  if (e != CMSD_OK || batch == 0) return e;
  e = bind_pass_workspace(a, workspace, workspace_bytes, cmsd_logit_pass_fused_workspace_bytes(batch, k_max, vocab));
  if (e != CMSD_OK) return e;
  const int es = dtype == CMSD_F32 ? 4 : 2;
  const int64_t rows = (int64_t)batch * (2 * k_max + 1);
  if (!launch_fits(rows, kFusedBD)) return CMSD_ERR_ARG;
  const int S = verify_slices(vocab, es);
  SlicePart* ws = static_cast<SlicePart*>(workspace);
  // the counters end the workspace (its size rounded down to 4 bytes): calls of any
  // batch that fits share them, clear of the slice records and row slots at its start
  int32_t* cnt = reinterpret_cast<int32_t*>(static_cast<char*>(workspace) + (workspace_bytes & ~(size_t)3)) - batch;
  const hipStream_t st = as_stream(stream);
  if (dtype == CMSD_F32)
    hipLaunchKernelGGL((k_fused_pass<float>), dim3((unsigned)rows), dim3(kFusedBD), 0, st, a, S, ws, cnt);
  else
    hipLaunchKernelGGL((k_fused_pass<Bf16>), dim3((unsigned)rows), dim3(kFusedBD), 0, st, a, S, ws, cnt);
  return launched();
}

}  // extern "C"
