// Router scores s_i = Router(t_i) (Sec. 4.2): linear router + softmax over
// all experts.
//
// bf16: logits = x Wr^T on the matrix cores (v_mfma_f32_16x16x32_bf16, fp32
// accumulation; a bf16 x bf16 product is exact in fp32).  A workgroup owns a
// 32-token x 32-expert tile of one of S slices of the hidden dimension; its
// four waves split the slice in quarters and issue all their operand loads
// at once, and the partial tiles are summed in wave order through LDS.  With
// few tokens (a decode step) the hidden dimension is split over S <= 4
// workgroups so that more CUs share the router matrix; the S partial logits
// go to the workspace and the softmax sums them in slice order, so the result
// does not depend on scheduling.
// f32: one thread per (token, expert) dot product.
// Softmax: one wave per token row; all partial loads of a pass are issued
// together and the row is staged in LDS (one read pass, one write pass).
// Optionally the kernel also stores x in the chunk-major layout the expert
// FFN reads ([H/c][T][c], c elements per 16-byte chunk): the workgroups of the
// first expert tile already hold every 16-byte chunk of x in registers.
#include <algorithm>

#include "route_dev.h"

namespace dmoe {
namespace {

using dev::kMaxSplits;

constexpr int kRouterTile = 32;
constexpr int kRouterSteps = 8;  // K steps of 32 per load burst

__global__ __launch_bounds__(256) void router_logits_bf16_kernel(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ w, int T, int H, int E, int S,
    float* __restrict__ part, bf16_t* __restrict__ xk) {
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int q = lane >> 4;   // k-group of the MFMA operand / row group of the result
  const int c = lane & 15;   // row of A (token) / column of B (expert)
  const int t0 = blockIdx.x * kRouterTile;
  const int e0 = blockIdx.y * kRouterTile;
  const int slice = H / S;
  const int kw = slice >> 2;
  const int kbeg = blockIdx.z * slice + wave * kw;
  const int steps = kw >> 5;

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

  for (int sc = 0; sc < steps; sc += kRouterSteps) {
    const int ns = min(kRouterSteps, steps - sc);
    bf16x8 a[kRouterSteps][2], b[kRouterSteps][2];
#pragma unroll
    for (int s = 0; s < kRouterSteps; ++s)
      if (s < ns)
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          a[s][r] = ld_bf16x8(pa[r] + (sc + s) * 32);
          b[s][r] = ld_bf16x8(pb[r] + (sc + s) * 32);
        }
#pragma unroll
    for (int s = 0; s < kRouterSteps; ++s)
      if (s < ns)
#pragma unroll
        for (int r = 0; r < 2; ++r)
#pragma unroll
          for (int u = 0; u < 2; ++u)
            acc[r][u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[s][r], b[s][u], acc[r][u], 0, 0, 0);
    if (xk && blockIdx.y == 0) {
      // chunk (kbeg + 32*(sc+s))/8 + q of token t0 + 16r + c
#pragma unroll
      for (int s = 0; s < kRouterSteps; ++s)
        if (s < ns)
#pragma unroll
          for (int r = 0; r < 2; ++r) {
            const int t = t0 + r * 16 + c;
            const int j = ((kbeg + (sc + s) * 32) >> 3) + q;
            if (t < T)
              *reinterpret_cast<bf16x8*>(xk + (static_cast<size_t>(j) * T + t) * 8) = a[s][r];
          }
    }
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
  float* out = part + static_cast<size_t>(blockIdx.z) * T * E;
#pragma unroll
  for (int r = 0; r < 2; ++r) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      f32x4 v = acc[r][s];
#pragma unroll
      for (int ww = 0; ww < 3; ++ww) v += red[ww][r * 2 + s][lane];
      const int e = e0 + s * 16 + c;
      if (e >= E) continue;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = t0 + r * 16 + q * 4 + i;
        if (t < T) out[static_cast<size_t>(t) * E + e] = v[i];
      }
    }
  }
}

// fp32 router: grid (ceil(E / 16), T).  Wave w of a workgroup computes the
// logits of experts 16*bx + w, + 4, ... for token t: each lane accumulates
// the features h = lane, lane + 64, ... of x[t] . w[e] (coalesced row reads),
// then the wave sums its lanes in a fixed order (dev::wave_sum).
constexpr int kF32RouterExperts = 16;

__global__ __launch_bounds__(256) void router_logits_f32_kernel(
    const float* __restrict__ x, const float* __restrict__ w, int T, int H, int E,
    float* __restrict__ part, float* __restrict__ xk) {
  const int t = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const float* xr = x + static_cast<size_t>(t) * H;
  if (xk && blockIdx.x == 0)
    for (int h = threadIdx.x; h < H; h += blockDim.x) xk[(static_cast<size_t>(h >> 2) * T + t) * 4 + (h & 3)] = xr[h];
  const int e1 = min(E, static_cast<int>(blockIdx.x + 1) * kF32RouterExperts);
  for (int e = blockIdx.x * kF32RouterExperts + wave; e < e1; e += 4) {
    const float* wr = w + static_cast<size_t>(e) * H;
    float acc = 0.f;
    for (int h = lane; h < H; h += kWave) acc = fmaf(xr[h], wr[h], acc);
    acc = dev::wave_sum(acc);
    if (lane == 0) part[static_cast<size_t>(t) * E + e] = acc;
  }
}

// One wave per token row, four rows per workgroup.  Up to 512 experts the
// row is reduced in registers (dev::softmax_loaded, the routine the fused
// routing kernel uses); wider rows are staged in LDS (dynamic: 4*E floats).
// part may alias probs (S == 1): a row is read whole before it is written.
template <int NQ>
__global__ __launch_bounds__(256) void softmax_rows_reg_kernel(const float* part, int S,
                                                               const float* __restrict__ bias, int T, int E,
                                                               float* probs, float* logits) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  dev::RowPartials<NQ> r[1];
  dev::load_row<NQ>(part, static_cast<size_t>(T) * E, S, bias, E, t, r[0]);
  const bool live[1] = {true};
  float* const out[1] = {probs + static_cast<size_t>(t) * E};
  float* const lds[1] = {nullptr};
  float* const lo[1] = {logits ? logits + static_cast<size_t>(t) * E : nullptr};
  dev::softmax_loaded<NQ, 1>(r, live, S, bias != nullptr, E, out, lds, lo);
}

__global__ __launch_bounds__(256) void softmax_rows_kernel(const float* part, int S,
                                                           const float* __restrict__ bias, int T,
                                                           int E, float* probs, float* logits) {
  extern __shared__ float zrow[];
  const int wave = threadIdx.x >> 6;
  const int t = blockIdx.x * 4 + wave;
  if (t >= T) return;
  dev::softmax_row(part + static_cast<size_t>(t) * E, static_cast<size_t>(T) * E, S, bias, E,
                   zrow + static_cast<size_t>(wave) * E, probs + static_cast<size_t>(t) * E,
                   logits ? logits + static_cast<size_t>(t) * E : nullptr);
}

// Slices of the hidden dimension: enough router workgroups to spread the
// router matrix over about half the CUs, each slice a multiple of 128.
int router_splits(int T, int H, int E) {
  const long tiles = static_cast<long>((T + kRouterTile - 1) / kRouterTile) * ((E + kRouterTile - 1) / kRouterTile);
  int S = 1;
  while (S < kMaxSplits && tiles * S < 128 && (H / 128) % (2 * S) == 0) S *= 2;
  return S;
}
}  // namespace

size_t router_workspace_bytes(int T, int H, int E, dmoe_dtype dt) {
  if (dt != DMOE_BF16) return 0;
  const int S = router_splits(T, H, E);
  return S > 1 ? static_cast<size_t>(S) * T * E * sizeof(float) : 0;
}

hipError_t launch_router_partials(const void* x, const void* w, dmoe_dtype dt, int T, int H, int E,
                                  float* probs, void* x_chunked, void* workspace, size_t ws_bytes,
                                  hipStream_t s, float** part_out, int* S_out) {
  int S = 1;
  float* part = probs;  // S == 1: the logits go to probs, read back in place by the softmax
  if (dt == DMOE_BF16) {
    const size_t need = router_workspace_bytes(T, H, E, dt);
    if (need > 0 && workspace && ws_bytes >= need) {
      S = router_splits(T, H, E);
      part = static_cast<float*>(workspace);
    }
    dim3 grid((T + kRouterTile - 1) / kRouterTile, (E + kRouterTile - 1) / kRouterTile, S);
    router_logits_bf16_kernel<<<grid, 256, 0, s>>>(static_cast<const bf16_t*>(x),
                                                    static_cast<const bf16_t*>(w), T, H, E, S, part,
                                                    static_cast<bf16_t*>(x_chunked));
  } else {
    dim3 grid((E + kF32RouterExperts - 1) / kF32RouterExperts, T);
    router_logits_f32_kernel<<<grid, 256, 0, s>>>(static_cast<const float*>(x),
                                                   static_cast<const float*>(w), T, H, E, part,
                                                   static_cast<float*>(x_chunked));
  }
  *part_out = part;
  *S_out = S;
  return hipGetLastError();
}

hipError_t launch_router(const void* x, const void* w, const float* bias, dmoe_dtype dt, int T,
                         int H, int E, float* logits, float* probs, void* x_chunked,
                         void* workspace, size_t ws_bytes, hipStream_t s) {
  float* part = nullptr;
  int S = 1;
  hipError_t err = launch_router_partials(x, w, dt, T, H, E, probs, x_chunked, workspace, ws_bytes, s,
                                          &part, &S);
  if (err != hipSuccess) return err;
  const unsigned blocks = (T + 3) / 4;
  if (E <= 256) {
    softmax_rows_reg_kernel<1><<<blocks, 256, 0, s>>>(part, S, bias, T, E, probs, logits);
  } else if (E <= dev::kRegSoftmaxMaxE) {
    softmax_rows_reg_kernel<2><<<blocks, 256, 0, s>>>(part, S, bias, T, E, probs, logits);
  } else {
    const size_t lds = static_cast<size_t>(4) * E * sizeof(float);
    softmax_rows_kernel<<<blocks, 256, lds, s>>>(part, S, bias, T, E, probs, logits);
  }
  return hipGetLastError();
}

}  // namespace dmoe
