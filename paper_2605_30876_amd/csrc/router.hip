// Router scores s_i = Router(t_i) (Sec. 4.2): linear router + softmax over
// all experts.
//
// bf16: logits = x Wr^T on the matrix cores (v_mfma_f32_16x16x32_bf16, fp32
// accumulation; a bf16 x bf16 product is exact in fp32).  A workgroup owns a
// 32-token x 32-expert tile; its four waves split the hidden dimension in
// quarters and the partial tiles are summed in wave order through LDS, so the
// result does not depend on scheduling.
// f32: one thread per (token, expert) dot product.
// Softmax: one wave per token row, max-subtracted, in place when the caller
// does not keep the logits.
#include "dmoe_common.h"

namespace dmoe {
namespace {

constexpr int kRouterTile = 32;

__global__ __launch_bounds__(256) void router_logits_bf16_kernel(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ w, const float* __restrict__ bias,
    int T, int H, int E, float* __restrict__ logits) {
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int q = lane >> 4;   // k-group of the MFMA operand / row group of the result
  const int c = lane & 15;   // row of A (token) / column of B (expert)
  const int t0 = blockIdx.x * kRouterTile;
  const int e0 = blockIdx.y * kRouterTile;
  const int kw = H >> 2;
  const int kbeg = wave * kw;

  const bf16_t* pa[2];
  const bf16_t* pb[2];
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    // ragged token / expert tails: clamp the rows read, skip the writes
    const int t = min(t0 + r * 16 + c, T - 1);
    const int e = min(e0 + r * 16 + c, E - 1);
    pa[r] = x + static_cast<size_t>(t) * H + kbeg + q * 8;
    pb[r] = w + static_cast<size_t>(e) * H + kbeg + q * 8;
  }
  f32x4 acc[2][2];
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int s = 0; s < 2; ++s) acc[r][s] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int k0 = 0; k0 < kw; k0 += 32) {
    bf16x8 a0 = ld_bf16x8(pa[0] + k0), a1 = ld_bf16x8(pa[1] + k0);
    bf16x8 b0 = ld_bf16x8(pb[0] + k0), b1 = ld_bf16x8(pb[1] + k0);
    acc[0][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, b0, acc[0][0], 0, 0, 0);
    acc[0][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, b1, acc[0][1], 0, 0, 0);
    acc[1][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, b0, acc[1][0], 0, 0, 0);
    acc[1][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, b1, acc[1][1], 0, 0, 0);
  }

  __shared__ f32x4 red[3][4][kWave];
  if (wave > 0) {
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int s = 0; s < 2; ++s) red[wave - 1][r * 2 + s][lane] = acc[r][s];
  }
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int r = 0; r < 2; ++r) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      f32x4 v = acc[r][s];
#pragma unroll
      for (int ww = 0; ww < 3; ++ww) v += red[ww][r * 2 + s][lane];
      const int e = e0 + s * 16 + c;
      if (e >= E) continue;
      const float b = bias ? bias[e] : 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = t0 + r * 16 + q * 4 + i;
        if (t < T) logits[static_cast<size_t>(t) * E + e] = v[i] + b;
      }
    }
  }
}

__global__ __launch_bounds__(256) void router_logits_f32_kernel(
    const float* __restrict__ x, const float* __restrict__ w, const float* __restrict__ bias,
    int T, int H, int E, float* __restrict__ logits) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  const int t = blockIdx.y;
  if (e >= E) return;
  const float* xr = x + static_cast<size_t>(t) * H;
  const float* wr = w + static_cast<size_t>(e) * H;
  float acc = 0.f;
  for (int h = 0; h < H; ++h) acc = fmaf(xr[h], wr[h], acc);
  logits[static_cast<size_t>(t) * E + e] = acc + (bias ? bias[e] : 0.f);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m));
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
  return v;
}

// One wave per token row; z and p may alias (in-place softmax).
__global__ __launch_bounds__(256) void softmax_rows_kernel(const float* z, int T, int E, float* p) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const float* zr = z + static_cast<size_t>(t) * E;
  float* pr = p + static_cast<size_t>(t) * E;
  float m = -INFINITY;
  for (int e = lane; e < E; e += kWave) m = fmaxf(m, zr[e]);
  m = wave_max(m);
  float s = 0.f;
  for (int e = lane; e < E; e += kWave) s += expf(zr[e] - m);
  s = wave_sum(s);
  for (int e = lane; e < E; e += kWave) pr[e] = expf(zr[e] - m) / s;
}

}  // namespace

hipError_t launch_router(const void* x, const void* w, const float* bias, dmoe_dtype dt, int T,
                         int H, int E, float* logits, float* probs, hipStream_t s) {
  float* z = logits ? logits : probs;
  if (dt == DMOE_BF16) {
    dim3 grid((T + kRouterTile - 1) / kRouterTile, (E + kRouterTile - 1) / kRouterTile);
    router_logits_bf16_kernel<<<grid, 256, 0, s>>>(static_cast<const bf16_t*>(x),
                                                    static_cast<const bf16_t*>(w), bias, T, H, E, z);
  } else {
    dim3 grid((E + 255) / 256, T);
    router_logits_f32_kernel<<<grid, 256, 0, s>>>(static_cast<const float*>(x),
                                                   static_cast<const float*>(w), bias, T, H, E, z);
  }
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  softmax_rows_kernel<<<(T + 3) / 4, 256, 0, s>>>(z, T, E, probs);
  return hipGetLastError();
}

}  // namespace dmoe
