// Expert execution: the SwiGLU FFN of every unique expert of the forward over
// the rows that selected it, plus the always-on shared expert over all tokens.
//
//   h    = silu(Wg x) * (Wu x)        gate/up kernel  -> h buffer (bf16 / f32)
//   out  = Wd h                       down kernel     -> slot_out[t][j] / shared_out[t]
//
// Work is indexed by (weight-row tile, group): group u < max_unique is the
// u-th unique routed expert (groups past the device-side n_unique exit at
// once), the last group is the shared expert.  A workgroup streams its
// weight tile from HBM once and applies it to every row of its group, so each
// selected expert's weights are read once per forward.
//
// bf16 path (matrix cores, v_mfma_f32_16x16x32_bf16, fp32 accumulation):
//  * A operand = weight rows, B operand = token rows, C = [weight row][token].
//  * gate/up: a 16-row A tile interleaves gate and up rows of 8 intermediate
//    units so that every lane's four accumulators are (g_i, g_i+1, u_i, u_i+1)
//    of one token: SwiGLU is applied in registers, no exchange needed.
//  * the four waves of a workgroup split the reduction (K) dimension in
//    quarters; partial tiles are summed in wave order through LDS, so results
//    are identical from run to run.
//  * a lane's 8-element K group is the same index set in A and B, which is all
//    the matrix instruction needs; each 16-byte load covers 64 contiguous
//    bytes of a row across the four lane groups.
// f32 path: plain per-thread dot products (small fp32 layers).
#include <algorithm>
#include <numeric>

#include "dmoe_common.h"

namespace dmoe {
namespace {

struct Group {
  int r0;         // first row of the group in the row space (h buffer row)
  int n;          // rows (tokens) in the group
  int expert;     // routed expert id, or -1 for the shared expert
  const int* tok;  // token of each row (routed) or nullptr (row c is token c)
};

__device__ __forceinline__ bool decode_group(int gidx, int max_unique, const int* n_unique,
                                             const int* unique, const int* offsets,
                                             const int* row_token, int T, int Tk, Group& g) {
  if (gidx < max_unique) {
    if (gidx >= *n_unique) return false;
    g.expert = unique[gidx];
    g.r0 = offsets[gidx];
    g.n = offsets[gidx + 1] - g.r0;
    g.tok = row_token + g.r0;
  } else {
    g.expert = -1;
    g.r0 = Tk;
    g.n = T;
    g.tok = nullptr;
  }
  return g.n > 0;
}

constexpr int kThreads = 256;

template <int NT, int U>
__global__ __launch_bounds__(kThreads) void ffn_gateup_bf16_kernel(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ wg, const bf16_t* __restrict__ wu,
    const bf16_t* __restrict__ wsg, const bf16_t* __restrict__ wsu,
    const int* __restrict__ n_unique, const int* __restrict__ unique,
    const int* __restrict__ offsets, const int* __restrict__ row_token, int T, int H, int I,
    int I_s, int Tk, int max_unique, int ldh, bf16_t* __restrict__ hbuf) {
  Group g;
  if (!decode_group(blockIdx.y, max_unique, n_unique, unique, offsets, row_token, T, Tk, g)) return;
  const int Iw = g.expert >= 0 ? I : I_s;
  const int i0 = blockIdx.x * 16;
  if (i0 >= Iw) return;
  const bf16_t* Wg = g.expert >= 0 ? wg + static_cast<size_t>(g.expert) * I * H : wsg;
  const bf16_t* Wu = g.expert >= 0 ? wu + static_cast<size_t>(g.expert) * I * H : wsu;

  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int q = lane >> 4;
  const int c = lane & 15;
  const int kw = H >> 2;
  const int kbeg = wave * kw;

  // A-row c of tile rt: gate or up row of intermediate unit i0 + rt*8 + 2*(c/4) + c%2.
  const bf16_t* pa[2];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    const int i = i0 + rt * 8 + 2 * (c >> 2) + (c & 1);
    pa[rt] = ((c & 2) ? Wu : Wg) + static_cast<size_t>(i) * H + kbeg + q * 8;
  }

  __shared__ f32x4 red[3][2 * NT][kWave];
  for (int p0 = 0; p0 < g.n; p0 += 16 * NT) {
    const bf16_t* pb[NT];
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) {
      const int col = min(p0 + ct * 16 + c, g.n - 1);
      const int tok = g.tok ? g.tok[col] : col;
      pb[ct] = x + static_cast<size_t>(tok) * H + kbeg + q * 8;
    }
    f32x4 acc[2][NT];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int ct = 0; ct < NT; ++ct) acc[rt][ct] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int k0 = 0; k0 < kw; k0 += 32 * U) {
      bf16x8 a[U][2], b[U][NT];
#pragma unroll
      for (int u = 0; u < U; ++u) {
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) a[u][rt] = ld_bf16x8(pa[rt] + k0 + u * 32);
#pragma unroll
        for (int ct = 0; ct < NT; ++ct) b[u][ct] = ld_bf16x8(pb[ct] + k0 + u * 32);
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int ct = 0; ct < NT; ++ct)
            acc[rt][ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u][rt], b[u][ct], acc[rt][ct], 0, 0, 0);
    }

    if (wave > 0) {
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int ct = 0; ct < NT; ++ct) red[wave - 1][rt * NT + ct][lane] = acc[rt][ct];
    }
    __syncthreads();
    if (wave == 0) {
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
#pragma unroll
        for (int ct = 0; ct < NT; ++ct) {
          f32x4 v = acc[rt][ct];
#pragma unroll
          for (int ww = 0; ww < 3; ++ww) v += red[ww][rt * NT + ct][lane];
          const int col = p0 + ct * 16 + c;
          if (col < g.n) {
            const uint32_t h0 = f32_to_bf16(silu_f32(v[0]) * v[2]);
            const uint32_t h1 = f32_to_bf16(silu_f32(v[1]) * v[3]);
            bf16_t* dst = hbuf + static_cast<size_t>(g.r0 + col) * ldh + i0 + rt * 8 + 2 * q;
            *reinterpret_cast<uint32_t*>(dst) = h0 | (h1 << 16);
          }
        }
      }
    }
    __syncthreads();
  }
}

template <int NT, int U>
__global__ __launch_bounds__(kThreads) void ffn_down_bf16_kernel(
    const bf16_t* __restrict__ wd, const bf16_t* __restrict__ wsd,
    const int* __restrict__ n_unique, const int* __restrict__ unique,
    const int* __restrict__ offsets, const int* __restrict__ row_token,
    const int* __restrict__ row_slot, int T, int H, int I, int I_s, int k, int Tk, int max_unique,
    int ldh, const bf16_t* __restrict__ hbuf, float* __restrict__ slot_out,
    float* __restrict__ shared_out) {
  Group g;
  if (!decode_group(blockIdx.y, max_unique, n_unique, unique, offsets, row_token, T, Tk, g)) return;
  const int Kd = g.expert >= 0 ? I : I_s;
  const bf16_t* Wd = g.expert >= 0 ? wd + static_cast<size_t>(g.expert) * H * I : wsd;
  const int j0 = blockIdx.x * 32;

  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int q = lane >> 4;
  const int c = lane & 15;
  const int kw = Kd >> 2;
  const int kbeg = wave * kw;

  const bf16_t* pa[2];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) pa[rt] = Wd + static_cast<size_t>(j0 + rt * 16 + c) * Kd + kbeg + q * 8;

  __shared__ f32x4 red[3][2 * NT][kWave];
  for (int p0 = 0; p0 < g.n; p0 += 16 * NT) {
    const bf16_t* pb[NT];
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) {
      const int col = min(p0 + ct * 16 + c, g.n - 1);
      pb[ct] = hbuf + static_cast<size_t>(g.r0 + col) * ldh + kbeg + q * 8;
    }
    f32x4 acc[2][NT];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int ct = 0; ct < NT; ++ct) acc[rt][ct] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int k0 = 0; k0 < kw; k0 += 32 * U) {
      bf16x8 a[U][2], b[U][NT];
#pragma unroll
      for (int u = 0; u < U; ++u) {
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) a[u][rt] = ld_bf16x8(pa[rt] + k0 + u * 32);
#pragma unroll
        for (int ct = 0; ct < NT; ++ct) b[u][ct] = ld_bf16x8(pb[ct] + k0 + u * 32);
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int ct = 0; ct < NT; ++ct)
            acc[rt][ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u][rt], b[u][ct], acc[rt][ct], 0, 0, 0);
    }

    if (wave > 0) {
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int ct = 0; ct < NT; ++ct) red[wave - 1][rt * NT + ct][lane] = acc[rt][ct];
    }
    __syncthreads();
    if (wave == 0) {
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
#pragma unroll
        for (int ct = 0; ct < NT; ++ct) {
          f32x4 v = acc[rt][ct];
#pragma unroll
          for (int ww = 0; ww < 3; ++ww) v += red[ww][rt * NT + ct][lane];
          const int col = p0 + ct * 16 + c;
          if (col < g.n) {
            const int j = j0 + rt * 16 + 4 * q;
            float* dst;
            if (g.tok) {
              const int r = g.r0 + col;
              dst = slot_out + (static_cast<size_t>(row_token[r]) * k + row_slot[r]) * H + j;
            } else {
              dst = shared_out + static_cast<size_t>(col) * H + j;
            }
            *reinterpret_cast<f32x4*>(dst) = v;
          }
        }
      }
    }
    __syncthreads();
  }
}

// ---- f32 path -------------------------------------------------------------

__global__ __launch_bounds__(kThreads) void ffn_gateup_f32_kernel(
    const float* __restrict__ x, const float* __restrict__ wg, const float* __restrict__ wu,
    const float* __restrict__ wsg, const float* __restrict__ wsu, const int* __restrict__ n_unique,
    const int* __restrict__ unique, const int* __restrict__ offsets,
    const int* __restrict__ row_token, int T, int H, int I, int I_s, int Tk, int max_unique,
    int ldh, float* __restrict__ hbuf) {
  Group g;
  if (!decode_group(blockIdx.y, max_unique, n_unique, unique, offsets, row_token, T, Tk, g)) return;
  const int Iw = g.expert >= 0 ? I : I_s;
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i >= Iw) return;
  const float* wgr = (g.expert >= 0 ? wg + static_cast<size_t>(g.expert) * I * H : wsg) + static_cast<size_t>(i) * H;
  const float* wur = (g.expert >= 0 ? wu + static_cast<size_t>(g.expert) * I * H : wsu) + static_cast<size_t>(i) * H;
  for (int col = 0; col < g.n; ++col) {
    const int tok = g.tok ? g.tok[col] : col;
    const float* xr = x + static_cast<size_t>(tok) * H;
    float a = 0.f, b = 0.f;
    for (int h = 0; h < H; ++h) {
      a = fmaf(xr[h], wgr[h], a);
      b = fmaf(xr[h], wur[h], b);
    }
    hbuf[static_cast<size_t>(g.r0 + col) * ldh + i] = silu_f32(a) * b;
  }
}

__global__ __launch_bounds__(kThreads) void ffn_down_f32_kernel(
    const float* __restrict__ wd, const float* __restrict__ wsd, const int* __restrict__ n_unique,
    const int* __restrict__ unique, const int* __restrict__ offsets,
    const int* __restrict__ row_token, const int* __restrict__ row_slot, int T, int H, int I,
    int I_s, int k, int Tk, int max_unique, int ldh, const float* __restrict__ hbuf,
    float* __restrict__ slot_out, float* __restrict__ shared_out) {
  Group g;
  if (!decode_group(blockIdx.y, max_unique, n_unique, unique, offsets, row_token, T, Tk, g)) return;
  const int Kd = g.expert >= 0 ? I : I_s;
  const int j = blockIdx.x * kThreads + threadIdx.x;
  if (j >= H) return;
  const float* wr = (g.expert >= 0 ? wd + static_cast<size_t>(g.expert) * H * I : wsd) + static_cast<size_t>(j) * Kd;
  for (int col = 0; col < g.n; ++col) {
    const float* hr = hbuf + static_cast<size_t>(g.r0 + col) * ldh;
    float acc = 0.f;
    for (int i = 0; i < Kd; ++i) acc = fmaf(hr[i], wr[i], acc);
    if (g.tok) {
      const int r = g.r0 + col;
      slot_out[(static_cast<size_t>(row_token[r]) * k + row_slot[r]) * H + j] = acc;
    } else {
      shared_out[static_cast<size_t>(col) * H + j] = acc;
    }
  }
}

// Largest unroll U in {4, 2, 1} with kw a multiple of 32*U.
int pick_unroll(int kw) { return kw % 128 == 0 ? 4 : (kw % 64 == 0 ? 2 : 1); }

// Token columns per pass: enough 16-wide tiles for the expected rows of a
// routed expert (T*k spread over max_unique experts), at most 4.
int pick_ntiles(int T, int k, int max_unique) {
  const long rows = (static_cast<long>(T) * k + max_unique - 1) / max_unique;
  return rows <= 16 ? 1 : (rows <= 32 ? 2 : 4);
}

#define DMOE_GU_ARGS                                                                             \
  static_cast<const bf16_t*>(a.x), static_cast<const bf16_t*>(a.wg),                             \
      static_cast<const bf16_t*>(a.wu), static_cast<const bf16_t*>(a.wsg),                       \
      static_cast<const bf16_t*>(a.wsu), a.sched.n_unique, a.sched.unique, a.sched.offsets,      \
      a.sched.row_token, a.T, a.H, a.I, a.I_s, Tk, a.max_unique, ldh,                            \
      static_cast<bf16_t*>(a.hbuf)
#define DMOE_DN_ARGS                                                                             \
  static_cast<const bf16_t*>(a.wd), static_cast<const bf16_t*>(a.wsd), a.sched.n_unique,        \
      a.sched.unique, a.sched.offsets, a.sched.row_token, a.sched.row_slot, a.T, a.H, a.I, a.I_s, \
      a.k, Tk, a.max_unique, ldh, static_cast<const bf16_t*>(a.hbuf), a.slot_out, a.shared_out

template <int NT>
void launch_bf16_nt(const FfnArgs& a, int Tk, int ldh, dim3 g_gu, dim3 g_dn, hipStream_t s) {
  switch (pick_unroll(a.H >> 2)) {
    case 4: ffn_gateup_bf16_kernel<NT, 4><<<g_gu, kThreads, 0, s>>>(DMOE_GU_ARGS); break;
    case 2: ffn_gateup_bf16_kernel<NT, 2><<<g_gu, kThreads, 0, s>>>(DMOE_GU_ARGS); break;
    default: ffn_gateup_bf16_kernel<NT, 1><<<g_gu, kThreads, 0, s>>>(DMOE_GU_ARGS); break;
  }
  // One unroll serves both K = I (routed) and K = I_s (shared): pick it for
  // their greatest common divisor.
  const int kd = a.I_s > 0 ? std::gcd(a.I, a.I_s) : a.I;
  switch (pick_unroll(kd >> 2)) {
    case 4: ffn_down_bf16_kernel<NT, 4><<<g_dn, kThreads, 0, s>>>(DMOE_DN_ARGS); break;
    case 2: ffn_down_bf16_kernel<NT, 2><<<g_dn, kThreads, 0, s>>>(DMOE_DN_ARGS); break;
    default: ffn_down_bf16_kernel<NT, 1><<<g_dn, kThreads, 0, s>>>(DMOE_DN_ARGS); break;
  }
}

}  // namespace

size_t ffn_hbuf_bytes(int T, int I, int I_s, int k, dmoe_dtype dt) {
  const size_t rows = static_cast<size_t>(T) * k + (I_s > 0 ? T : 0);
  const size_t ldh = static_cast<size_t>(std::max(I, I_s));
  return rows * ldh * (dt == DMOE_F32 ? 4 : 2);
}

hipError_t launch_ffn(const FfnArgs& a, dmoe_dtype dt, hipStream_t s) {
  const int Tk = a.T * a.k;
  const int ldh = std::max(a.I, a.I_s);
  const int groups = a.max_unique + (a.I_s > 0 ? 1 : 0);
  if (dt == DMOE_BF16) {
    dim3 g_gu(ldh / 16, groups), g_dn(a.H / 32, groups);
    switch (pick_ntiles(a.T, a.k, a.max_unique)) {
      case 1: launch_bf16_nt<1>(a, Tk, ldh, g_gu, g_dn, s); break;
      case 2: launch_bf16_nt<2>(a, Tk, ldh, g_gu, g_dn, s); break;
      default: launch_bf16_nt<4>(a, Tk, ldh, g_gu, g_dn, s); break;
    }
    return hipGetLastError();
  }
  dim3 g_gu((ldh + kThreads - 1) / kThreads, groups), g_dn((a.H + kThreads - 1) / kThreads, groups);
  ffn_gateup_f32_kernel<<<g_gu, kThreads, 0, s>>>(
      static_cast<const float*>(a.x), static_cast<const float*>(a.wg), static_cast<const float*>(a.wu),
      static_cast<const float*>(a.wsg), static_cast<const float*>(a.wsu), a.sched.n_unique,
      a.sched.unique, a.sched.offsets, a.sched.row_token, a.T, a.H, a.I, a.I_s, Tk, a.max_unique, ldh,
      static_cast<float*>(a.hbuf));
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  ffn_down_f32_kernel<<<g_dn, kThreads, 0, s>>>(
      static_cast<const float*>(a.wd), static_cast<const float*>(a.wsd), a.sched.n_unique,
      a.sched.unique, a.sched.offsets, a.sched.row_token, a.sched.row_slot, a.T, a.H, a.I, a.I_s,
      a.k, Tk, a.max_unique, ldh, static_cast<const float*>(a.hbuf), a.slot_out, a.shared_out);
  return hipGetLastError();
}

}  // namespace dmoe
