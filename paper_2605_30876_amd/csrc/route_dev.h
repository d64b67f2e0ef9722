// Device routines shared by the routing kernels (router softmax, block and
// token top-k, unique-expert schedule) and the fused small-forward routing
// kernel, so that every path computes bit-identical results.  Internal.
#pragma once

#include "dmoe_common.h"

namespace dmoe {
namespace dev {

// ---- wave reductions on the DPP network ------------------------------------
// quad_perm xor 1, xor 2, half-row mirror, row mirror, row_bcast15 (into rows
// 1 and 3), row_bcast31 (into rows 2 and 3): lane 63 ends with the reduction
// of all 64 lanes, which readlane broadcasts.  A fixed pattern of VALU data
// movement (no LDS crossbar round trips), so the result is deterministic.
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140,
              kDppBcast15 = 0x142, kDppBcast31 = 0x143;

// Lanes of rows outside ROWS keep `old`.
template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ int dpp(int old, int v) {
  return __builtin_amdgcn_update_dpp(old, v, CTRL, ROWS, 0xF, false);
}
template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ float dppf(float old, float v) {
  return __builtin_bit_cast(float, dpp<CTRL, ROWS>(__builtin_bit_cast(int, old), __builtin_bit_cast(int, v)));
}
__device__ __forceinline__ float lane63f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dppf<kDppXor1>(v, v));
  v = fmaxf(v, dppf<kDppXor2>(v, v));
  v = fmaxf(v, dppf<kDppHalfMirror>(v, v));
  v = fmaxf(v, dppf<kDppMirror>(v, v));
  v = fmaxf(v, dppf<kDppBcast15, 0xA>(v, v));
  v = fmaxf(v, dppf<kDppBcast31, 0xC>(v, v));
  return lane63f(v);
}

// Sum of the 64 lanes in a fixed tree order (rows outside a broadcast add 0).
__device__ __forceinline__ float wave_sum(float v) {
  v += dppf<kDppXor1>(0.f, v);
  v += dppf<kDppXor2>(0.f, v);
  v += dppf<kDppHalfMirror>(0.f, v);
  v += dppf<kDppMirror>(0.f, v);
  v += dppf<kDppBcast15, 0xA>(0.f, v);
  v += dppf<kDppBcast31, 0xC>(0.f, v);
  return lane63f(v);
}

constexpr int kMaxSplits = 4;  // router slices of the hidden dimension

// Logit of one element: the S partial sums p[0..S) in slice order, then the
// bias value bv when there is a bias.
__device__ __forceinline__ float sum_partials(const float (&p)[kMaxSplits], int S, bool has_bias, float bv) {
  float v = p[0];
#pragma unroll
  for (int s = 1; s < kMaxSplits; ++s)
    if (s < S) v += p[s];
  if (has_bias) v += bv;
  return v;
}

// Softmax of a row of logits z[0..E) (LDS) by one wave, max-subtracted:
// out (global) and z receive the probabilities, lo (global, optional) the
// logits.  Each lane handles e = lane, lane + 64, ... in that order.
__device__ inline void softmax_finish(float* z, int E, float* out, float* lo) {
  const int lane = threadIdx.x & 63;
  float m = -INFINITY;
  for (int e = lane; e < E; e += kWave) m = fmaxf(m, z[e]);
  m = wave_max(m);
  float sum = 0.f;
  for (int e = lane; e < E; e += kWave) sum += expf(z[e] - m);
  sum = wave_sum(sum);
  for (int e = lane; e < E; e += kWave) {
    const float v = z[e];
    const float pv = expf(v - m) / sum;
    out[e] = pv;
    z[e] = pv;
    if (lo) lo[e] = v;
  }
}

// Softmax of one token row from S partial logit planes + bias, by one wave;
// z is an LDS row of E floats.  A lane handles 4 elements (e = lane + 64*u)
// per pass and issues all their partial loads together.
__device__ inline void softmax_row(const float* pr, size_t plane, int S, const float* bias, int E,
                                   float* z, float* out, float* lo) {
  const int lane = threadIdx.x & 63;
  for (int e0 = 0; e0 < E; e0 += 4 * kWave) {
    float p[4][kMaxSplits], bv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = e0 + u * kWave + lane;
#pragma unroll
      for (int s = 0; s < kMaxSplits; ++s)
        if (s < S && e < E) p[u][s] = pr[s * plane + e];
      bv[u] = (bias && e < E) ? bias[e] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = e0 + u * kWave + lane;
      if (e < E) z[e] = sum_partials(p[u], S, bias != nullptr, bv[u]);
    }
  }
  softmax_finish(z, E, out, lo);
}

// ---- register softmax for E <= 256*NQ ---------------------------------------
// exp(z - m) as 2^(z*log2(e) - m*log2(e)) on the hardware exp2 (a few ulp;
// the argument is <= 0, so no overflow), and one reciprocal per row instead
// of a division per element.
constexpr float kLog2e = 1.4426950408889634f;
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// A wave owns a row; lane l holds elements e = 256*q + 4*l + c (q < NQ,
// c < 4), loaded as float4 when rows are 16-byte aligned (E % 4 == 0).
constexpr int kRegSoftmaxMaxE = 512;

template <int NQ>
struct RowPartials {
  f32x4 p[NQ][kMaxSplits];
  f32x4 b[NQ];
};

// Issue the loads of row t's S partial planes (and bias) for this lane.
template <int NQ>
__device__ __forceinline__ void load_row(const float* part, size_t plane, int S, const float* bias, int E, int t,
                                         RowPartials<NQ>& r) {
  const int lane = threadIdx.x & 63;
  const bool vec = (E & 3) == 0;
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int e0 = 256 * q + 4 * lane;
#pragma unroll
    for (int s = 0; s < kMaxSplits; ++s) {
      if (s >= S) continue;
      const float* src = part + s * plane + static_cast<size_t>(t) * E + e0;
      if (vec && e0 < E) {
        r.p[q][s] = *reinterpret_cast<const f32x4*>(src);
      } else {
#pragma unroll
        for (int c = 0; c < 4; ++c) r.p[q][s][c] = e0 + c < E ? src[c] : 0.f;
      }
    }
    if (bias) {
      if (vec && e0 < E) {
        r.b[q] = *reinterpret_cast<const f32x4*>(bias + e0);
      } else {
#pragma unroll
        for (int c = 0; c < 4; ++c) r.b[q][c] = e0 + c < E ? bias[e0 + c] : 0.f;
      }
    }
  }
}

// Softmax of RB loaded rows, stage by stage across the rows so that their
// dependent chains (wave reductions, exponentials) overlap.  For
// row u: out[u] (global) and, when given, lds[u] receive the probabilities,
// lo[u] (global, optional) the logits; rows with live[u] false are skipped.
// Each lane sums its own exponentials in (q, c) order, then the wave sum
// combines lanes: the arithmetic of a row does not depend on RB.
template <int NQ, int RB>
__device__ __forceinline__ void softmax_loaded(const RowPartials<NQ> (&r)[RB], const bool (&live)[RB], int S,
                                               bool has_bias, int E, float* const (&out)[RB],
                                               float* const (&lds)[RB], float* const (&lo)[RB]) {
  const int lane = threadIdx.x & 63;
  const bool vec = (E & 3) == 0;
  float z[RB][NQ][4];
  float m[RB];
#pragma unroll
  for (int u = 0; u < RB; ++u) {
    m[u] = -INFINITY;
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int e = 256 * q + 4 * lane + c;
        float v = r[u].p[q][0][c];
#pragma unroll
        for (int s = 1; s < kMaxSplits; ++s)
          if (s < S) v += r[u].p[q][s][c];
        if (has_bias) v += r[u].b[q][c];
        z[u][q][c] = v;
        if (e < E) m[u] = fmaxf(m[u], v);
      }
  }
#pragma unroll
  for (int u = 0; u < RB; ++u) m[u] = wave_max(m[u]);
  float ex[RB][NQ][4];
  float sum[RB];
#pragma unroll
  for (int u = 0; u < RB; ++u) {
    sum[u] = 0.f;
    const float ml = m[u] * kLog2e;
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int e = 256 * q + 4 * lane + c;
        ex[u][q][c] = exp2_hw(fmaf(z[u][q][c], kLog2e, -ml));
        if (e < E) sum[u] += ex[u][q][c];
      }
  }
#pragma unroll
  for (int u = 0; u < RB; ++u) sum[u] = __builtin_amdgcn_rcpf(wave_sum(sum[u]));  // 1 / sum
#pragma unroll
  for (int u = 0; u < RB; ++u) {
    if (!live[u]) continue;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int e0 = 256 * q + 4 * lane;
      if (e0 >= E) continue;
      f32x4 pv;
#pragma unroll
      for (int c = 0; c < 4; ++c) pv[c] = ex[u][q][c] * sum[u];
      if (vec) {
        *reinterpret_cast<f32x4*>(out[u] + e0) = pv;
        if (lds[u]) *reinterpret_cast<f32x4*>(lds[u] + e0) = pv;
        if (lo[u]) *reinterpret_cast<f32x4*>(lo[u] + e0) = f32x4{z[u][q][0], z[u][q][1], z[u][q][2], z[u][q][3]};
      } else {
#pragma unroll
        for (int c = 0; c < 4; ++c)
          if (e0 + c < E) {
            out[u][e0 + c] = pv[c];
            if (lds[u]) lds[u][e0 + c] = pv[c];
            if (lo[u]) lo[u][e0 + c] = z[u][q][c];
          }
      }
    }
  }
}

// ---- top-k in (score desc, id asc) order ------------------------------------
//
// Scores are ranked by order-preserving integer keys: a float's key orders
// like the float compare (-0 and +0 share a key, as they compare equal), and
// every float, NaN included, has one.  So each ranking below is a total
// order and a selection is always k distinct ids, whatever the scores hold
// (a NaN probability from a NaN hidden state still selects valid experts).

constexpr int kMaxK = 64;
constexpr int kNone = 0x7fffffff;

__device__ __forceinline__ uint32_t order_key(float f) {
  const uint32_t b = __float_as_uint(f + 0.0f);  // -0 -> +0: keys order like the float compare
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// The float a key came from (-0 comes back as +0, which compares equal).
__device__ __forceinline__ float key_value(uint32_t key) {
  return __uint_as_float((key & 0x80000000u) ? (key & 0x7FFFFFFFu) : ~key);
}

// (key a, id i) ranks before (key b, id j): higher key, then lower id.
__device__ __forceinline__ bool key_before(uint32_t a, int i, uint32_t b, int j) {
  return a > b || (a == b && i < j);
}

struct Cand {
  uint32_t key;  // order key of the score
  int i;         // expert id
};
// Sentinels: every candidate ranks after kCandTop and before kCandNone.
constexpr Cand kCandTop = {0xFFFFFFFFu, -1};
constexpr Cand kCandNone = {0u, kNone};

// Best candidate of the wave in (score desc, id asc) order; every lane gets it.
__device__ __forceinline__ void best_step(Cand& c, int ok, int oi) {
  const uint32_t k = static_cast<uint32_t>(ok);
  if (key_before(k, oi, c.key, c.i)) {
    c.key = k;
    c.i = oi;
  }
}
__device__ __forceinline__ Cand wave_best(Cand c) {
  int k = static_cast<int>(c.key);
  best_step(c, dpp<kDppXor1>(k, k), dpp<kDppXor1>(c.i, c.i));
  k = static_cast<int>(c.key);
  best_step(c, dpp<kDppXor2>(k, k), dpp<kDppXor2>(c.i, c.i));
  k = static_cast<int>(c.key);
  best_step(c, dpp<kDppHalfMirror>(k, k), dpp<kDppHalfMirror>(c.i, c.i));
  k = static_cast<int>(c.key);
  best_step(c, dpp<kDppMirror>(k, k), dpp<kDppMirror>(c.i, c.i));
  k = static_cast<int>(c.key);
  best_step(c, dpp<kDppBcast15, 0xA>(k, k), dpp<kDppBcast15, 0xA>(c.i, c.i));
  k = static_cast<int>(c.key);
  best_step(c, dpp<kDppBcast31, 0xC>(k, k), dpp<kDppBcast31, 0xC>(c.i, c.i));
  return Cand{static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(c.key), 63)),
              __builtin_amdgcn_readlane(c.i, 63)};
}

// The first `rounds` elements of row[0..E) (LDS) in order, by one wave: round
// r picks the best element strictly after round r-1's pick.  Lane 0 writes
// sel[r], selv[r].
__device__ inline void wave_topk(const float* row, int E, int rounds, int* sel, float* selv) {
  const int lane = threadIdx.x & 63;
  Cand prev = kCandTop;
  for (int r = 0; r < rounds; ++r) {
    Cand best = kCandNone;
    for (int e = lane; e < E; e += kWave) {
      const uint32_t k = order_key(row[e]);
      if (key_before(prev.key, prev.i, k, e) && key_before(k, e, best.key, best.i)) best = Cand{k, e};
    }
    best = wave_best(best);
    if (lane == 0) {
      sel[r] = best.i;
      selv[r] = key_value(best.key);
    }
    prev = best;
  }
}

constexpr int kRadixMaxPerLane = 16;  // E <= 1024

__device__ __forceinline__ uint32_t umin32(uint32_t a, uint32_t b) { return a < b ? a : b; }

// Minimum over the 64 lanes (same DPP pattern as wave_max).
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
  int x = static_cast<int>(v);
  x = static_cast<int>(umin32(x, dpp<kDppXor1>(x, x)));
  x = static_cast<int>(umin32(x, dpp<kDppXor2>(x, x)));
  x = static_cast<int>(umin32(x, dpp<kDppHalfMirror>(x, x)));
  x = static_cast<int>(umin32(x, dpp<kDppMirror>(x, x)));
  x = static_cast<int>(umin32(x, dpp<kDppBcast15, 0xA>(x, x)));
  x = static_cast<int>(umin32(x, dpp<kDppBcast31, 0xC>(x, x)));
  return static_cast<uint32_t>(__builtin_amdgcn_readlane(x, 63));
}

__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0));
}

// NJ values per lane (E <= 64*NJ): lane l holds e = 64*j + l.  RB rows are
// searched together (their bit loops are independent chains); rows with
// live[u] false are skipped (every row pointer must still be readable over
// [0, E): all loads are issued unconditionally, then masked, so they are in
// flight together).  With kMasked, only elements with inside[e] != 0 (LDS
// flags) take part, and each row must hold at least `rounds` of them.  live
// must be uniform over the wave.  See wave_topk_radix for the method.
template <int NJ, int RB, bool kMasked = false>
__device__ inline void wave_topk_radix_rows(const float* const (&row)[RB], const bool (&live)[RB], int E,
                                            int rounds, int* const (&sel)[RB], float* const (&selv)[RB],
                                            float* buf_v, int* buf_i, const int* inside = nullptr) {
  const int lane = threadIdx.x & 63;
  bool lv[RB];  // live, as a wave-uniform (scalar) value
#pragma unroll
  for (int u = 0; u < RB; ++u) lv[u] = __builtin_amdgcn_readfirstlane(live[u] ? 1 : 0) != 0;
  float val[RB][NJ];
  int flag[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int e = min(j * kWave + lane, E - 1);
    flag[j] = kMasked ? inside[e] : 1;
#pragma unroll
    for (int u = 0; u < RB; ++u) val[u][j] = row[u][e];
  }
  uint32_t key[RB][NJ];
#pragma unroll
  for (int u = 0; u < RB; ++u)
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const bool in = lv[u] && j * kWave + lane < E && flag[j] != 0;
      // excluded lanes: key 0, below every real key (real keys are >= 1)
      key[u][j] = in ? max(order_key(val[u][j]), 1u) : 0u;
    }
  // MSB-first search for the rounds-th largest key.  A row stops as soon as
  // exactly `rounds` keys are >= its prefix: the answer is then the smallest
  // of them (rows whose rounds-th and next keys are equal run all 32 bits).
  uint32_t prefix[RB];
  bool exact[RB];
#pragma unroll
  for (int u = 0; u < RB; ++u) {
    prefix[u] = 0;
    exact[u] = !lv[u];
  }
  for (int bit = 31; bit >= 0; --bit) {
    bool all = true;
#pragma unroll
    for (int u = 0; u < RB; ++u) {
      if (!exact[u]) {
        const uint32_t cand = prefix[u] | (1u << bit);
        int cnt = 0;
#pragma unroll
        for (int j = 0; j < NJ; ++j) cnt += __popcll(__ballot(key[u][j] >= cand));
        prefix[u] = cnt >= rounds ? cand : prefix[u];
        exact[u] = cnt == rounds;
      }
      all = all && exact[u];
    }
    if (all) break;
  }
#pragma unroll
  for (int u = 0; u < RB; ++u) {
    if (!lv[u] || !exact[u]) continue;
    uint32_t m = 0xFFFFFFFFu;
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if (key[u][j] >= prefix[u]) m = umin32(m, key[u][j]);
    prefix[u] = wave_min_u32(m);
  }
  // prefix[u] is now row u's rounds-th largest key; gather and rank row by row
#pragma unroll
  for (int u = 0; u < RB; ++u) {
    if (!lv[u]) continue;
    int n_gt = 0;
#pragma unroll
    for (int j = 0; j < NJ; ++j) n_gt += __popcll(__ballot(key[u][j] > prefix[u]));
    const int need_eq = rounds - n_gt;
    int eq_taken = 0, placed = 0;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const bool eq = key[u][j] == prefix[u];
      const uint64_t eq_mask = __ballot(eq);
      const bool take = key[u][j] > prefix[u] || (eq && eq_taken + lanes_below(eq_mask) < need_eq);
      eq_taken += __popcll(eq_mask);
      const uint64_t t_mask = __ballot(take);
      if (take) {
        const int pos = placed + lanes_below(t_mask);
        const int e = j * kWave + lane;
        buf_v[pos] = __uint_as_float(key[u][j]);  // the key's bits
        buf_i[pos] = e;
      }
      placed += __popcll(t_mask);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (rounds <= kWave) {
      // one gathered element per lane; ranks from broadcasts of the others
      const uint32_t kv = lane < rounds ? __float_as_uint(buf_v[lane]) : 0u;
      const int i = lane < rounds ? buf_i[lane] : kNone;
      int r = 0;
      for (int m = 0; m < rounds; ++m)
        r += key_before(static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(kv), m)),
                        __builtin_amdgcn_readlane(i, m), kv, i) ? 1 : 0;
      if (lane < rounds) {
        sel[u][r] = i;
        selv[u][r] = key_value(kv);
      }
    } else {
      for (int l = lane; l < rounds; l += kWave) {
        const uint32_t kv = __float_as_uint(buf_v[l]);
        const int i = buf_i[l];
        int r = 0;
        for (int m = 0; m < rounds; ++m) r += key_before(__float_as_uint(buf_v[m]), buf_i[m], kv, i) ? 1 : 0;
        sel[u][r] = i;
        selv[u][r] = key_value(kv);
      }
    }
    // the gather buffer is reused by the next row
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

template <int NJ>
__device__ inline void wave_topk_radix_n(const float* row, int E, int rounds, int* sel, float* selv, float* buf_v,
                                         int* buf_i) {
  const float* const rows[1] = {row};
  const bool live[1] = {true};
  int* const sels[1] = {sel};
  float* const selvs[1] = {selv};
  wave_topk_radix_rows<NJ, 1>(rows, live, E, rounds, sels, selvs, buf_v, buf_i);
}

// Top `rounds` of row[0..E) (LDS, E <= 64*kRadixMaxPerLane) by one wave, in
// (score desc, id asc) order, by radix selection: an MSB-first search over
// order-preserving integer keys finds the rounds-th largest key (each bit is
// one ballot count per register); the elements above it, then the lowest ids
// equal to it, are gathered in id order into buf_v (their keys' bits) / buf_i
// (LDS, rounds entries) and ranked among themselves by key and id.  Lanes write sel[r], selv[r].
__device__ inline void wave_topk_radix(const float* row, int E, int rounds, int* sel, float* selv, float* buf_v,
                                       int* buf_i) {
  if (E <= 64)
    wave_topk_radix_n<1>(row, E, rounds, sel, selv, buf_v, buf_i);
  else if (E <= 128)
    wave_topk_radix_n<2>(row, E, rounds, sel, selv, buf_v, buf_i);
  else if (E <= 256)
    wave_topk_radix_n<4>(row, E, rounds, sel, selv, buf_v, buf_i);
  else if (E <= 512)
    wave_topk_radix_n<8>(row, E, rounds, sel, selv, buf_v, buf_i);
  else
    wave_topk_radix_n<16>(row, E, rounds, sel, selv, buf_v, buf_i);
}

// ---- unique-expert schedule (one workgroup of kSchedThreads) ---------------

constexpr int kSchedThreads = 512;
constexpr int kMaskWords = kSchedThreads / 32;

constexpr int pad4(int E) { return (E + 3) & ~3; }

// LDS ints the schedule needs for E experts: cnt, base, run [E'], masks
// [E'][kMaskWords] (16-byte aligned rows), entry positions [kSchedThreads].
constexpr size_t schedule_lds_ints(int E) {
  return static_cast<size_t>(pad4(E)) * (3 + kMaskWords) + kSchedThreads;
}

// Inclusive prefix sum over the wave: shifts of 1, 2, 4, 8 within rows of 16
// lanes, then row 0 into row 1 and row 2 into row 3, then rows 0-1 into rows
// 2-3 (lanes reading outside their row add 0).
__device__ __forceinline__ int wave_incl_scan(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, true);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, true);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, true);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, true);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, kDppBcast15, 0xA, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, kDppBcast31, 0xC, 0xF, false);
  return v;
}

// Totals of the schedule from the per-expert selection counts (thread e of
// the kSchedThreads passes c = the count of expert e, 0 for e >= E; E <=
// kSchedThreads): ascending unique ids, their row offsets, n_unique, the
// work items and n_work; base[e] (LDS or global) receives expert e's first
// row.  Called by all threads of the workgroup.
__device__ inline void schedule_totals(int c, int gs, int E, const dmoe_schedule& sched, int* base) {
  __shared__ int wrows[kSchedThreads / kWave];
  __shared__ int wuniq[kSchedThreads / kWave];
  __shared__ int wchunk[kSchedThreads / kWave];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int rows = c * gs;
  const int pres = c > 0 ? 1 : 0;
  const int chunks = (rows + DMOE_WORK_ROWS - 1) / DMOE_WORK_ROWS;  // work items of this expert
  const int r_incl = wave_incl_scan(rows);
  const int u_incl = wave_incl_scan(pres);
  const int c_incl = wave_incl_scan(chunks);
  if (lane == kWave - 1) {
    wrows[wave] = r_incl;
    wuniq[wave] = u_incl;
    wchunk[wave] = c_incl;
  }
  __syncthreads();
  int r_off = 0, u_off = 0, c_off = 0;
  for (int w = 0; w < wave; ++w) {
    r_off += wrows[w];
    u_off += wuniq[w];
    c_off += wchunk[w];
  }
  const int r_excl = r_off + r_incl - rows;
  const int u_excl = u_off + u_incl - pres;
  const int c_excl = c_off + c_incl - chunks;
  if (tid < E) {
    base[tid] = r_excl;
    if (pres) {
      sched.unique[u_excl] = tid;
      sched.offsets[u_excl] = r_excl;
    }
    int4* work = reinterpret_cast<int4*>(sched.work) + c_excl;
    for (int q = 0; q < chunks; ++q)
      work[q] = make_int4(tid, r_excl + q * DMOE_WORK_ROWS, min(DMOE_WORK_ROWS, rows - q * DMOE_WORK_ROWS), q);
  }
  if (tid == kSchedThreads - 1) {
    sched.offsets[u_excl + pres] = r_excl + rows;
    *sched.n_unique = u_excl + pres;
    *sched.n_work = c_excl + chunks;
  }
}

// Builds the schedule of n_groups expert lists of k (experts: global or LDS,
// [n_groups][k]; group g covers tokens g*gs .. g*gs+gs-1).  Called by all
// kSchedThreads threads of the workgroup; lds holds schedule_lds_ints(E) ints
// (16-byte aligned).
//   1. counts the selections of every expert (LDS integer atomics),
//   2. scans the counts: ascending unique ids, their row offsets, n_unique,
//   3. places the (group, slot) entries in rounds of kSchedThreads, in index
//      order: an entry's rank among earlier entries of its expert is a
//      running count plus the entries below it in the round's per-expert
//      bitmask (read as four 128-bit words), so each expert's rows come out
//      in token order and the schedule is identical on every run; then all
//      threads write the round's rows.  With place_rows false step 3 is left
//      to a many-workgroup launch (schedule_rows_kernel).
__device__ inline void schedule_wg(const int32_t* experts, int n_groups, int gs, int k, int E, int* lds,
                                   const dmoe_schedule& sched, bool place_rows = true) {
  int32_t* const row_token = sched.row_token;
  int32_t* const row_slot = sched.row_slot;
  const int Ep = pad4(E);
  int* cnt = lds;                                          // [E] selections
  int* base = cnt + Ep;                                    // [E] first row
  int* run = base + Ep;                                    // [E] entries placed so far
  unsigned* mask = reinterpret_cast<unsigned*>(run + Ep);  // [E][kMaskWords]
  int* pos = reinterpret_cast<int*>(mask + static_cast<size_t>(Ep) * kMaskWords);  // [kSchedThreads]

  const int tid = threadIdx.x;
  for (int e = tid; e < E; e += kSchedThreads) {
    cnt[e] = 0;
    run[e] = 0;
    uint4* m4 = reinterpret_cast<uint4*>(mask + e * kMaskWords);
#pragma unroll
    for (int w = 0; w < kMaskWords / 4; ++w) m4[w] = make_uint4(0u, 0u, 0u, 0u);
  }
  __syncthreads();

  const int n_entries = n_groups * k;
  for (int i = tid; i < n_entries; i += kSchedThreads) {
    const int e = experts[i];
    if (e >= 0 && e < E) atomicAdd(&cnt[e], 1);
  }
  __syncthreads();

  schedule_totals(tid < E ? cnt[tid] : 0, gs, E, sched, base);
  __syncthreads();
  if (!place_rows) return;

  const int word = tid >> 5;
  const unsigned bit = 1u << (tid & 31);
  for (int r0 = 0; r0 < n_entries; r0 += kSchedThreads) {
    const int i = r0 + tid;
    const int e = i < n_entries ? experts[i] : -1;
    const bool active = e >= 0 && e < E;
    if (active) atomicOr(&mask[e * kMaskWords + word], bit);
    __syncthreads();
    bool last = true;
    int below = 0;
    if (active) {
      const uint4* m4 = reinterpret_cast<const uint4*>(mask + e * kMaskWords);
      unsigned m[kMaskWords];
#pragma unroll
      for (int w = 0; w < kMaskWords / 4; ++w) {
        const uint4 q = m4[w];
        m[4 * w] = q.x;
        m[4 * w + 1] = q.y;
        m[4 * w + 2] = q.z;
        m[4 * w + 3] = q.w;
      }
#pragma unroll
      for (int w = 0; w < kMaskWords; ++w) {
        if (w < word) below += __popc(m[w]);
        if (w > word && m[w]) last = false;
        if (w == word) {
          below += __popc(m[w] & (bit - 1u));
          if (m[w] & ~(bit | (bit - 1u))) last = false;
        }
      }
      pos[tid] = base[e] + (run[e] + below) * gs;
    } else {
      pos[tid] = -1;  // an id outside [0, E): no rows
    }
    __syncthreads();
    if (active) {
      if (last) run[e] += below + 1;
      atomicAnd(&mask[e * kMaskWords + word], ~bit);
    }
    // rows of the round's entries, written by all threads
    const int n_round = min(kSchedThreads, n_entries - r0);
    for (int idx = tid; idx < n_round * gs; idx += kSchedThreads) {
      const int ie = idx / gs, tl = idx - ie * gs;
      const int ig = r0 + ie;
      const int g = ig / k;
      const int p = pos[ie];
      if (p < 0) continue;
      row_token[p + tl] = g * gs + tl;
      row_slot[p + tl] = ig - g * k;
    }
    __syncthreads();
  }
}

// The schedule of a single group (one block): its k distinct experts in
// ascending id order, each with all gs rows of the group, slot = the expert's
// position in the group's list, and their work items.  The same schedule
// schedule_wg builds for n_groups == 1.  Called by all threads of the
// workgroup (k <= kWave); lds holds kWave ints.
__device__ inline void schedule_one_group(const int32_t* experts, int gs, int k, int* lds,
                                          const dmoe_schedule& sched) {
  int* slot_of = lds;  // [k] slot of the rank-u expert
  const int tid = threadIdx.x;
  const int chunks = (gs + DMOE_WORK_ROWS - 1) / DMOE_WORK_ROWS;  // work items per expert
  if (tid < kWave) {
    const int e = tid < k ? experts[tid] : 0x7fffffff;
    int r = 0;
    for (int m = 0; m < k; ++m) r += __builtin_amdgcn_readlane(e, m) < e ? 1 : 0;
    if (tid < k) {
      slot_of[r] = tid;
      sched.unique[r] = e;
      sched.offsets[r] = r * gs;
      int4* work = reinterpret_cast<int4*>(sched.work) + r * chunks;
      for (int c = 0; c < chunks; ++c)
        work[c] = make_int4(e, r * gs + c * DMOE_WORK_ROWS, min(DMOE_WORK_ROWS, gs - c * DMOE_WORK_ROWS), c);
    }
    if (tid == 0) {
      sched.offsets[k] = k * gs;
      *sched.n_unique = k;
      *sched.n_work = k * chunks;
    }
  }
  __syncthreads();
  for (int i = tid; i < k * gs; i += blockDim.x) {
    const int u = i / gs;
    sched.row_token[i] = i - u * gs;
    sched.row_slot[i] = slot_of[u];
  }
}

}  // namespace dev
}  // namespace dmoe
