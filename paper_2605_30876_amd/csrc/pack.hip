// Layout conversions for the expert FFN.
//
// Expert weights (once per model load).  bf16 uses matrix-core fragment
// order: the A operand of v_mfma_f32_16x16x32_bf16 is a 16-row x 32-column
// tile in which lane l = 16*q + c holds row c, columns 8q .. 8q+7 (16 bytes).
// Storing each such tile as its 64 lane-ordered 16-byte pieces (1 KiB) makes a
// wave's operand load one contiguous 1 KiB read, and a run of K steps one
// contiguous burst.
//   gate/up  w13[e][it][ks][lane][8], it < I/8, ks < H/32: row c of tile it is
//            the gate (c%4 < 2) or up row of intermediate unit 8*it + 2*(c/4)
//            + c%2, so a result lane holds (g_i, g_i+1, u_i, u_i+1) of a token.
//   down     w2[e][jt][ks][lane][8], jt < H/16, ks < I/32: row c of tile jt is
//            output feature 16*jt + c.
// f32: reduction-major, so that consecutive lanes (consecutive output units)
// read consecutive weights: w13[e][h][u], u < 2I, is the gate (u < I) or up
// (u - I) weight of unit u at feature h; w2[e][i][j] = w_down[e][j][i].
//
// Activations: chunk-major [H/c][T][c] with c elements per 16-byte chunk
// (c = 8 for bf16, 4 for f32), so the 16 tokens of a matrix-core column tile
// read 256 contiguous bytes per chunk.
#include "dmoe_common.h"

namespace dmoe {
namespace {

constexpr int kPackThreads = 256;

unsigned blocks_for(size_t n) { return static_cast<unsigned>((n + kPackThreads - 1) / kPackThreads); }

// One thread per 16-byte piece of the packed gate/up tensor.
__global__ __launch_bounds__(kPackThreads) void pack_gateup_bf16_kernel(
    const bf16_t* __restrict__ wg, const bf16_t* __restrict__ wu, int E, int I, int H,
    bf16_t* __restrict__ out) {
  const size_t n = static_cast<size_t>(E) * (I / 8) * (H / 32) * 64;
  const size_t p = static_cast<size_t>(blockIdx.x) * kPackThreads + threadIdx.x;
  if (p >= n) return;
  const int lane = static_cast<int>(p & 63);
  size_t rest = p >> 6;
  const int ks = static_cast<int>(rest % (H / 32));
  rest /= (H / 32);
  const int it = static_cast<int>(rest % (I / 8));
  const size_t e = rest / (I / 8);
  const int q = lane >> 4, c = lane & 15;
  const int i = 8 * it + 2 * (c >> 2) + (c & 1);
  const bf16_t* src = ((c & 2) ? wu : wg) + (e * I + i) * H + 32 * ks + 8 * q;
  *reinterpret_cast<u16x8*>(out + p * 8) = *reinterpret_cast<const u16x8*>(src);
}

__global__ __launch_bounds__(kPackThreads) void pack_down_bf16_kernel(
    const bf16_t* __restrict__ wd, int E, int H, int I, bf16_t* __restrict__ out) {
  const size_t n = static_cast<size_t>(E) * (H / 16) * (I / 32) * 64;
  const size_t p = static_cast<size_t>(blockIdx.x) * kPackThreads + threadIdx.x;
  if (p >= n) return;
  const int lane = static_cast<int>(p & 63);
  size_t rest = p >> 6;
  const int ks = static_cast<int>(rest % (I / 32));
  rest /= (I / 32);
  const int jt = static_cast<int>(rest % (H / 16));
  const size_t e = rest / (H / 16);
  const int q = lane >> 4, c = lane & 15;
  const bf16_t* src = wd + (e * H + 16 * jt + c) * I + 32 * ks + 8 * q;
  *reinterpret_cast<u16x8*>(out + p * 8) = *reinterpret_cast<const u16x8*>(src);
}

// f32 gate/up: out[e][h][u] = u < I ? wg[e][u][h] : wu[e][u - I][h]; one
// thread per output element.
__global__ __launch_bounds__(kPackThreads) void stack_gateup_f32_kernel(
    const float* __restrict__ wg, const float* __restrict__ wu, int E, int I, int H,
    float* __restrict__ out) {
  const size_t per = static_cast<size_t>(I) * H;
  const size_t n = static_cast<size_t>(E) * 2 * per;
  const size_t p = static_cast<size_t>(blockIdx.x) * kPackThreads + threadIdx.x;
  if (p >= n) return;
  const size_t e = p / (2 * per), r = p % (2 * per);
  const size_t h = r / (2 * static_cast<size_t>(I)), u = r % (2 * static_cast<size_t>(I));
  out[p] = u < static_cast<size_t>(I) ? wg[e * per + u * H + h] : wu[e * per + (u - I) * H + h];
}

// f32 down: out[e][i][j] = wd[e][j][i]; one thread per output element.
__global__ __launch_bounds__(kPackThreads) void transpose_down_f32_kernel(const float* __restrict__ wd, int E,
                                                                          int H, int I, float* __restrict__ out) {
  const size_t per = static_cast<size_t>(H) * I;
  const size_t n = static_cast<size_t>(E) * per;
  const size_t p = static_cast<size_t>(blockIdx.x) * kPackThreads + threadIdx.x;
  if (p >= n) return;
  const size_t e = p / per, r = p % per;
  const size_t i = r / H, j = r % H;
  out[p] = wd[e * per + j * I + i];
}

// Row-major [T][nc] -> chunk-major [nc][T] of 16-byte chunks (nc chunks per
// row); one thread per chunk, consecutive threads on consecutive tokens.
__global__ __launch_bounds__(kPackThreads) void chunk_rows_kernel(const f32x4* __restrict__ x, int T, int nc,
                                                                  f32x4* __restrict__ out) {
  const size_t n = static_cast<size_t>(T) * nc;
  const size_t p = static_cast<size_t>(blockIdx.x) * kPackThreads + threadIdx.x;
  if (p >= n) return;
  const size_t j = p / T, t = p % T;
  out[p] = x[t * nc + j];
}

}  // namespace

hipError_t launch_pack_weights(const void* wg, const void* wu, const void* wd, dmoe_dtype dt, int E,
                               int H, int I, void* w13, void* w2, hipStream_t s) {
  if (dt == DMOE_BF16) {
    const size_t n13 = static_cast<size_t>(E) * (I / 8) * (H / 32) * 64;
    pack_gateup_bf16_kernel<<<blocks_for(n13), kPackThreads, 0, s>>>(
        static_cast<const bf16_t*>(wg), static_cast<const bf16_t*>(wu), E, I, H,
        static_cast<bf16_t*>(w13));
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    const size_t nd = static_cast<size_t>(E) * (H / 16) * (I / 32) * 64;
    pack_down_bf16_kernel<<<blocks_for(nd), kPackThreads, 0, s>>>(static_cast<const bf16_t*>(wd), E, H, I,
                                                                  static_cast<bf16_t*>(w2));
    return hipGetLastError();
  }
  const size_t n13 = static_cast<size_t>(E) * 2 * I * H;
  stack_gateup_f32_kernel<<<blocks_for(n13), kPackThreads, 0, s>>>(
      static_cast<const float*>(wg), static_cast<const float*>(wu), E, I, H, static_cast<float*>(w13));
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const size_t nd = static_cast<size_t>(E) * H * I;
  transpose_down_f32_kernel<<<blocks_for(nd), kPackThreads, 0, s>>>(static_cast<const float*>(wd), E, H, I,
                                                                    static_cast<float*>(w2));
  return hipGetLastError();
}

hipError_t launch_pack_activations(const void* x, dmoe_dtype dt, int T, int H, void* x_chunked,
                                   hipStream_t s) {
  // both element types move whole 16-byte chunks (8 bf16 or 4 f32)
  const int nc = H / chunk_elems(dt);
  chunk_rows_kernel<<<blocks_for(static_cast<size_t>(T) * nc), kPackThreads, 0, s>>>(
      static_cast<const f32x4*>(x), T, nc, static_cast<f32x4*>(x_chunked));
  return hipGetLastError();
}

}  // namespace dmoe
