// Expert execution: the SwiGLU FFN of every unique expert of the forward over
// the rows that selected it, plus the always-on shared expert over all tokens.
//
//   h    = silu(Wg x) * (Wu x)        gate/up kernel -> h rows (workspace)
//   out  = Wd h                       down kernel    -> slot_out[t][j] / shared_out[t]
//
// Groups: g < n_unique is the g-th unique routed expert of the schedule; the
// shared expert is one more group.  A workgroup owns one 16-row weight tile
// of one group, streams it from HBM once and applies it to every row (token)
// of the group, so each selected expert's weights are read once per forward.
// The grid covers the largest possible group count; workgroups of groups past
// the device-side count exit at once.
//
// bf16 path (matrix cores, v_mfma_f32_16x16x32_bf16, fp32 accumulation):
//  * A operand = weight rows, B operand = token rows, C = [weight row][token].
//  * A gate/up tile interleaves the gate and up rows of 8 intermediate units,
//    so a lane's four accumulators are (g_i, g_i+1, u_i, u_i+1) of one token
//    and SwiGLU is applied in registers.
//  * Tiles of 16 weight rows give many small workgroups: a burst of weight
//    reads spread over several workgroups per CU keeps every HBM channel busy
//    and the CUs evenly loaded (32-row tiles left a third of the bandwidth
//    unused on small forwards).
//  * The four waves of a workgroup split the reduction dimension in quarters.
//    Each wave issues all of its weight loads at once (one burst per up to
//    KMAX 32-wide K steps), with the token operand double-buffered in chunks
//    behind it; partial tiles are summed in wave order through LDS, so
//    results do not depend on scheduling.
//  * A lane's 8-element K group is the same index set in A and B, which is all
//    the matrix instruction needs; the four lane groups of a 16-byte load
//    cover 64 contiguous bytes of a row.
// f32 path: plain per-thread dot products (small fp32 layers).
#include <algorithm>

#include "dmoe_common.h"

namespace dmoe {
namespace {

constexpr int kThreads = 256;

struct Group {
  int r0;          // first row of the group in the row space (h buffer row)
  int n;           // rows (tokens) in the group
  int expert;      // routed expert id, or -1 for the shared expert
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

// ---- bf16 kernels ----------------------------------------------------------

struct FfnParams {
  const bf16_t* x;
  const bf16_t* wg;
  const bf16_t* wu;
  const bf16_t* wd;
  const bf16_t* wsg;
  const bf16_t* wsu;
  const bf16_t* wsd;
  const int* n_unique;
  const int* unique;
  const int* offsets;
  const int* row_token;
  const int* row_slot;
  int T, H, I, I_s, k, Tk, ldh, max_unique;
  bf16_t* hbuf;
  float* slot_out;
  float* shared_out;
};

// Operands of one wave for up to KMAX K-steps (32 each) of its K-slice.
// A: one 16-row weight tile, all steps issued at once; B: NT 16-column token
// tiles, double-buffered in chunks of kBChunk steps.
constexpr int kBChunk = 4;

template <int NT, int KMAX>
struct WaveOps {
  bf16x8 a[KMAX];
  bf16x8 b[2][kBChunk][NT];
};

template <int NT, int KMAX>
__device__ __forceinline__ void issue_a(WaveOps<NT, KMAX>& w, const bf16_t* pa, int k0, int ns) {
#pragma unroll
  for (int s = 0; s < KMAX; ++s)
    if (s < ns) w.a[s] = ld_bf16x8(pa + k0 + s * 32);
}

template <int BUF, int NT, int KMAX>
__device__ __forceinline__ void issue_b(WaveOps<NT, KMAX>& w, const bf16_t* const* pb, int k0, int chunk, int ns) {
#pragma unroll
  for (int s = 0; s < kBChunk; ++s)
    if (chunk * kBChunk + s < ns)
#pragma unroll
      for (int ct = 0; ct < NT; ++ct) w.b[BUF][s][ct] = ld_bf16x8(pb[ct] + k0 + (chunk * kBChunk + s) * 32);
}

template <int C, int NT, int KMAX>
__device__ __forceinline__ void mma_chunk(WaveOps<NT, KMAX>& w, const bf16_t* const* pb, int k0, int ns,
                                          f32x4 (&acc)[NT]) {
  constexpr int NCH = KMAX / kBChunk;
  if constexpr (C < NCH) {
    if (C * kBChunk < ns) {
      if constexpr (C + 1 < NCH) issue_b<(C + 1) & 1>(w, pb, k0, C + 1, ns);
      __builtin_amdgcn_sched_barrier(0);  // keep the next chunk's loads where they are
#pragma unroll
      for (int s = 0; s < kBChunk; ++s)
        if (C * kBChunk + s < ns)
#pragma unroll
          for (int ct = 0; ct < NT; ++ct)
            acc[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w.a[C * kBChunk + s], w.b[C & 1][s][ct],
                                                              acc[ct], 0, 0, 0);
      mma_chunk<C + 1>(w, pb, k0, ns, acc);
    }
  }
}

// acc[ct] += A[k0 .. k0 + 32*steps) . B_ct[same]^T for this wave's slice, in
// bursts of KMAX steps: token chunk 0, the weight burst, then the chunks.
template <int NT, int KMAX>
__device__ __forceinline__ void wave_dot(const bf16_t* pa, const bf16_t* const* pb, int steps,
                                         f32x4 (&acc)[NT]) {
  WaveOps<NT, KMAX> w;
  for (int sc = 0; sc < steps; sc += KMAX) {
    const int ns = min(KMAX, steps - sc);
    issue_b<0>(w, pb, sc * 32, 0, ns);
    issue_a(w, pa, sc * 32, ns);
    __builtin_amdgcn_sched_barrier(0);
    mma_chunk<0>(w, pb, sc * 32, ns, acc);
  }
}

// Sum the four waves' partial tiles into wave 0's registers (wave order).
template <int NT>
__device__ __forceinline__ void reduce_waves(f32x4 (&acc)[NT], f32x4 (*red)[NT][kWave], int wave, int lane) {
  if (wave > 0) {
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) red[wave - 1][ct][lane] = acc[ct];
  }
  __syncthreads();
  if (wave == 0) {
#pragma unroll
    for (int ct = 0; ct < NT; ++ct)
#pragma unroll
      for (int ww = 0; ww < 3; ++ww) acc[ct] += red[ww][ct][lane];
  }
}

template <int NT>
__device__ __forceinline__ void zero(f32x4 (&acc)[NT]) {
#pragma unroll
  for (int ct = 0; ct < NT; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// grid (ldh / 8, groups): tile of 8 intermediate units (16 A rows).
template <int NT, int KMAX>
__global__ __launch_bounds__(kThreads) void ffn_gateup_bf16_kernel(FfnParams p) {
  Group g;
  if (!decode_group(blockIdx.y, p.max_unique, p.n_unique, p.unique, p.offsets, p.row_token, p.T, p.Tk, g))
    return;
  const int Iw = g.expert >= 0 ? p.I : p.I_s;
  const int i0 = blockIdx.x * 8;
  if (i0 >= Iw) return;
  const int H = p.H;
  const bf16_t* Wg = g.expert >= 0 ? p.wg + static_cast<size_t>(g.expert) * p.I * H : p.wsg;
  const bf16_t* Wu = g.expert >= 0 ? p.wu + static_cast<size_t>(g.expert) * p.I * H : p.wsu;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int q = lane >> 4, c = lane & 15;
  const int kw = H >> 2, kbeg = wave * kw, steps = kw >> 5;
  // A-row c: gate (c%4 < 2) or up row of intermediate unit i0 + 2*(c/4) + c%2.
  const int i = i0 + 2 * (c >> 2) + (c & 1);
  const bf16_t* pa = ((c & 2) ? Wu : Wg) + static_cast<size_t>(i) * H + kbeg + q * 8;

  __shared__ f32x4 red[3][NT][kWave];
  for (int p0 = 0; p0 < g.n; p0 += 16 * NT) {
    const bf16_t* pb[NT];
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) {
      const int col = min(p0 + ct * 16 + c, g.n - 1);
      const int tok = g.tok ? g.tok[col] : col;
      pb[ct] = p.x + static_cast<size_t>(tok) * H + kbeg + q * 8;
    }
    f32x4 acc[NT];
    zero(acc);
    wave_dot<NT, KMAX>(pa, pb, steps, acc);
    reduce_waves(acc, red, wave, lane);
    if (wave == 0) {
#pragma unroll
      for (int ct = 0; ct < NT; ++ct) {
        const int col = p0 + ct * 16 + c;
        if (col < g.n) {
          const f32x4 v = acc[ct];
          const uint32_t h0 = f32_to_bf16(silu_f32(v[0]) * v[2]);
          const uint32_t h1 = f32_to_bf16(silu_f32(v[1]) * v[3]);
          bf16_t* dst = p.hbuf + static_cast<size_t>(g.r0 + col) * p.ldh + i0 + 2 * q;
          *reinterpret_cast<uint32_t*>(dst) = h0 | (h1 << 16);
        }
      }
    }
    __syncthreads();  // red is reused by the next pass
  }
}

// grid (H / 16, groups): tile of 16 output features.
template <int NT, int KMAX>
__global__ __launch_bounds__(kThreads) void ffn_down_bf16_kernel(FfnParams p) {
  Group g;
  if (!decode_group(blockIdx.y, p.max_unique, p.n_unique, p.unique, p.offsets, p.row_token, p.T, p.Tk, g))
    return;
  const int Kd = g.expert >= 0 ? p.I : p.I_s;
  const int H = p.H;
  const bf16_t* Wd = g.expert >= 0 ? p.wd + static_cast<size_t>(g.expert) * H * p.I : p.wsd;
  const int j0 = blockIdx.x * 16;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int q = lane >> 4, c = lane & 15;
  const int kw = Kd >> 2, kbeg = wave * kw, steps = kw >> 5;
  const bf16_t* pa = Wd + static_cast<size_t>(j0 + c) * Kd + kbeg + q * 8;

  __shared__ f32x4 red[3][NT][kWave];
  for (int p0 = 0; p0 < g.n; p0 += 16 * NT) {
    const bf16_t* pb[NT];
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) {
      const int col = min(p0 + ct * 16 + c, g.n - 1);
      pb[ct] = p.hbuf + static_cast<size_t>(g.r0 + col) * p.ldh + kbeg + q * 8;
    }
    f32x4 acc[NT];
    zero(acc);
    wave_dot<NT, KMAX>(pa, pb, steps, acc);
    reduce_waves(acc, red, wave, lane);
    if (wave == 0) {
#pragma unroll
      for (int ct = 0; ct < NT; ++ct) {
        const int col = p0 + ct * 16 + c;
        if (col < g.n) {
          const int j = j0 + 4 * q;
          float* dst;
          if (g.tok) {
            const int r = g.r0 + col;
            dst = p.slot_out + (static_cast<size_t>(p.row_token[r]) * p.k + p.row_slot[r]) * H + j;
          } else {
            dst = p.shared_out + static_cast<size_t>(col) * H + j;
          }
          *reinterpret_cast<f32x4*>(dst) = acc[ct];
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

// ---- launch ---------------------------------------------------------------

// Token columns per pass: enough 16-wide tiles for the expected rows of a
// routed expert (T*k spread over max_unique experts), at most 4.
int pick_ntiles(int T, int k, int max_unique) {
  const long rows = (static_cast<long>(T) * k + max_unique - 1) / max_unique;
  return rows <= 16 ? 1 : (rows <= 32 ? 2 : 4);
}

template <int NT>
hipError_t launch_bf16(const FfnParams& p, int groups, hipStream_t s) {
  constexpr int KMAX = NT <= 2 ? 16 : 8;
  ffn_gateup_bf16_kernel<NT, KMAX><<<dim3(p.ldh / 8, groups), kThreads, 0, s>>>(p);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  ffn_down_bf16_kernel<NT, 8><<<dim3(p.H / 16, groups), kThreads, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace

size_t ffn_workspace_bytes(int T, int I, int I_s, int k, dmoe_dtype dt) {
  const size_t rows = static_cast<size_t>(T) * k + (I_s > 0 ? T : 0);
  const size_t ldh = static_cast<size_t>(std::max(I, I_s));
  return rows * ldh * (dt == DMOE_F32 ? 4 : 2);
}

hipError_t launch_ffn(const FfnArgs& a, dmoe_dtype dt, hipStream_t s) {
  const int Tk = a.T * a.k;
  const int ldh = std::max(a.I, a.I_s);
  const int groups = a.max_unique + (a.I_s > 0 ? 1 : 0);
  if (dt == DMOE_BF16) {
    FfnParams p{static_cast<const bf16_t*>(a.x), static_cast<const bf16_t*>(a.wg),
                static_cast<const bf16_t*>(a.wu), static_cast<const bf16_t*>(a.wd),
                static_cast<const bf16_t*>(a.wsg), static_cast<const bf16_t*>(a.wsu),
                static_cast<const bf16_t*>(a.wsd), a.sched.n_unique, a.sched.unique,
                a.sched.offsets, a.sched.row_token, a.sched.row_slot, a.T, a.H, a.I, a.I_s, a.k,
                Tk, ldh, a.max_unique, static_cast<bf16_t*>(a.workspace), a.slot_out, a.shared_out};
    switch (pick_ntiles(a.T, a.k, a.max_unique)) {
      case 1: return launch_bf16<1>(p, groups, s);
      case 2: return launch_bf16<2>(p, groups, s);
      default: return launch_bf16<4>(p, groups, s);
    }
  }
  void* hbuf = a.workspace;
  dim3 g_gu((ldh + kThreads - 1) / kThreads, groups), g_dn((a.H + kThreads - 1) / kThreads, groups);
  ffn_gateup_f32_kernel<<<g_gu, kThreads, 0, s>>>(
      static_cast<const float*>(a.x), static_cast<const float*>(a.wg), static_cast<const float*>(a.wu),
      static_cast<const float*>(a.wsg), static_cast<const float*>(a.wsu), a.sched.n_unique,
      a.sched.unique, a.sched.offsets, a.sched.row_token, a.T, a.H, a.I, a.I_s, Tk, a.max_unique, ldh,
      static_cast<float*>(hbuf));
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  ffn_down_f32_kernel<<<g_dn, kThreads, 0, s>>>(
      static_cast<const float*>(a.wd), static_cast<const float*>(a.wsd), a.sched.n_unique,
      a.sched.unique, a.sched.offsets, a.sched.row_token, a.sched.row_slot, a.T, a.H, a.I, a.I_s,
      a.k, Tk, a.max_unique, ldh, static_cast<const float*>(hbuf), a.slot_out, a.shared_out);
  return hipGetLastError();
}

}  // namespace dmoe
