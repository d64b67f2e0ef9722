// Wave-level helpers of the bf16 expert FFN kernels: packed weight tiles as
// the matrix-core A operand, chunk-major token rows as the B operand, bursts
// of K-steps with double-buffered token chunks, and the fixed-order sum of
// the four waves' partial tiles.  Internal; shared by ffn.hip and layer.hip.
#pragma once

#include "dmoe_common.h"

namespace dmoe {
namespace fdev {

constexpr int kFrag = 512;  // bf16 elements of one packed 16 x 32 weight tile (1 KiB)

// Operands of one wave for up to KMAX K-steps (32 each) of its K-slice.
// A: RT 16-row weight tiles, all steps issued at once; B: NT 16-column token
// tiles in chunks of BC steps, double-buffered when a burst has more than one
// chunk.  Each B fragment feeds RT matrix instructions.
template <int NT, int KMAX, int BC, int RT = 1>
struct WaveOps {
  static constexpr int kChunks = KMAX / BC;
  bf16x8 a[RT][KMAX];
  bf16x8 b[kChunks > 1 ? 2 : 1][BC][NT];
};

// A: packed tiles, step s of tile r at pa + r*tstride + s*kFrag (one
// contiguous burst per tile).  kStream: non-temporal loads, for weights no
// other workgroup of the launch reads again.
template <bool kStream, int NT, int KMAX, int BC, int RT>
__device__ __forceinline__ void issue_a(WaveOps<NT, KMAX, BC, RT>& w, const bf16_t* pa, size_t tstride, int ns) {
#pragma unroll
  for (int r = 0; r < RT; ++r)
#pragma unroll
    for (int s = 0; s < KMAX; ++s)
      if (s < ns)
        w.a[r][s] = kStream ? ld_bf16x8_stream(pa + r * tstride + s * kFrag) : ld_bf16x8(pa + r * tstride + s * kFrag);
}

// B: chunk-major rows, step s at pb[ct] + s*bstep.
template <int BUF, int NT, int KMAX, int BC, int RT>
__device__ __forceinline__ void issue_b(WaveOps<NT, KMAX, BC, RT>& w, const bf16_t* const* pb, int bstep, int chunk,
                                        int ns) {
#pragma unroll
  for (int s = 0; s < BC; ++s)
    if (chunk * BC + s < ns)
#pragma unroll
      for (int ct = 0; ct < NT; ++ct) w.b[BUF][s][ct] = ld_bf16x8(pb[ct] + (chunk * BC + s) * bstep);
}

template <int C, int NT, int KMAX, int BC, int RT>
__device__ __forceinline__ void mma_chunk(WaveOps<NT, KMAX, BC, RT>& w, const bf16_t* const* pb, int bstep, int ns,
                                          f32x4 (&acc)[RT][NT]) {
  constexpr int NCH = KMAX / BC;
  if constexpr (C < NCH) {
    if (C * BC < ns) {
      if constexpr (C + 1 < NCH) issue_b<(C + 1) & 1>(w, pb, bstep, C + 1, ns);
      __builtin_amdgcn_sched_barrier(0);  // keep the next chunk's loads where they are
#pragma unroll
      for (int s = 0; s < BC; ++s)
        if (C * BC + s < ns)
#pragma unroll
          for (int ct = 0; ct < NT; ++ct)
#pragma unroll
            for (int r = 0; r < RT; ++r)
              acc[r][ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w.a[r][C * BC + s], w.b[C & 1][s][ct], acc[r][ct],
                                                                   0, 0, 0);
      mma_chunk<C + 1>(w, pb, bstep, ns, acc);
    }
  }
}

// acc[ct] += A . B_ct^T over this wave's `steps` K-steps, in bursts of KMAX
// steps: token chunk 0, the weight burst, then the remaining token chunks.
// With a_held (the slice is one burst, steps <= KMAX, already in w.a from
// the previous pass over the same weights) the weights are not loaded again.
// kStream: the weights are loaded non-temporally (see issue_a).
template <bool kStream, int NT, int KMAX, int BC, int RT>
__device__ __forceinline__ void wave_dot(WaveOps<NT, KMAX, BC, RT>& w, const bf16_t* pa, size_t tstride,
                                         const bf16_t* const* pb, int bstep, int steps, f32x4 (&acc)[RT][NT],
                                         bool a_held) {
  for (int sc = 0; sc < steps; sc += KMAX) {
    const int ns = min(KMAX, steps - sc);
    const bf16_t* pbs[NT];
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) pbs[ct] = pb[ct] + sc * bstep;
    issue_b<0>(w, pbs, bstep, 0, ns);
    if (!a_held) issue_a<kStream>(w, pa + sc * kFrag, tstride, ns);
    __builtin_amdgcn_sched_barrier(0);
    mma_chunk<0>(w, pbs, bstep, ns, acc);
  }
}

// Sum the four waves' partial tiles into wave 0's registers (wave order).
template <int RT, int NT>
__device__ __forceinline__ void reduce_waves(f32x4 (&acc)[RT][NT], f32x4 (*red)[RT][NT][kWave], int wave,
                                             int lane) {
  if (wave > 0) {
#pragma unroll
    for (int r = 0; r < RT; ++r)
#pragma unroll
      for (int ct = 0; ct < NT; ++ct) red[wave - 1][r][ct][lane] = acc[r][ct];
  }
  __syncthreads();
  if (wave == 0) {
#pragma unroll
    for (int r = 0; r < RT; ++r)
#pragma unroll
      for (int ct = 0; ct < NT; ++ct)
#pragma unroll
        for (int ww = 0; ww < 3; ++ww) acc[r][ct] += red[ww][r][ct][lane];
  }
}

template <int RT, int NT>
__device__ __forceinline__ void zero(f32x4 (&acc)[RT][NT]) {
#pragma unroll
  for (int r = 0; r < RT; ++r)
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) acc[r][ct] = f32x4{0.f, 0.f, 0.f, 0.f};
}

}  // namespace fdev
}  // namespace dmoe
