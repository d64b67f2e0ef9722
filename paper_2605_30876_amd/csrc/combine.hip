// Weighted combine of the routed expert outputs and the shared expert:
//   y[t][h] = sum_j w[t][j] * slot_out[t][j][h] (+ shared_out[t][h])
// summed in slot order in fp32.  One thread per four consecutive outputs; a
// batch of slot rows is loaded at once (one memory round trip per batch).
// Slot outputs are float32 or scaled half (four fp16 values and the exponent
// byte of their 16-value group per thread and slot, decoded exactly to fp32).
// With a residual, res_out = res_in + y (the fp32 sum, rounded once to the
// residual's type) is written as well, for the next layer's input.
#include <type_traits>

#include "dmoe_common.h"

namespace dmoe {
namespace {

constexpr int kSlotBatch = 8;  // slot loads in flight together

__device__ __forceinline__ void store4(float* dst, const f32x4& v) { *reinterpret_cast<f32x4*>(dst) = v; }
__device__ __forceinline__ void store4(bf16_t* dst, const f32x4& v) {
  const uint32_t lo = f32_to_bf16(v[0]) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16);
  const uint32_t hi = f32_to_bf16(v[2]) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16);
  *reinterpret_cast<uint2*>(dst) = make_uint2(lo, hi);
}

constexpr int kCombineThreads = 64;  // small workgroups spread a decode step's combine over more CUs

__device__ __forceinline__ f32x4 load4(const float* p) { return *reinterpret_cast<const f32x4*>(p); }
__device__ __forceinline__ f32x4 load4(const bf16_t* p) {
  const uint2 u = *reinterpret_cast<const uint2*>(p);
  return f32x4{bf16_to_f32(static_cast<bf16_t>(u.x & 0xFFFFu)), bf16_to_f32(static_cast<bf16_t>(u.x >> 16)),
               bf16_to_f32(static_cast<bf16_t>(u.y & 0xFFFFu)), bf16_to_f32(static_cast<bf16_t>(u.y >> 16))};
}

// ResT: the residual's type, or void for none.
template <typename OutT, bool kF16S, typename ResT>
__global__ __launch_bounds__(kCombineThreads) void combine_kernel(const void* __restrict__ slot_out,
                                                      const float* __restrict__ w,
                                                      const float* __restrict__ shared_out, int T,
                                                      int H, int k, OutT* __restrict__ y,
                                                      const void* __restrict__ res_in,
                                                      void* __restrict__ res_out) {
  const int h4 = H >> 2;
  const size_t idx = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= static_cast<size_t>(T) * h4) return;
  const int t = static_cast<int>(idx / h4);
  const int hq = static_cast<int>(idx - static_cast<size_t>(t) * h4);  // group of four outputs
  const int h = hq * 4;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  const float* wt = w + static_cast<size_t>(t) * k;
  const size_t row0 = static_cast<size_t>(t) * k;  // slot row of (t, 0)
  const f32x4 sh = shared_out ? *reinterpret_cast<const f32x4*>(shared_out + static_cast<size_t>(t) * H + h)
                              : f32x4{0.f, 0.f, 0.f, 0.f};
  f32x4 rv = {0.f, 0.f, 0.f, 0.f};
  if constexpr (!std::is_void_v<ResT>) rv = load4(static_cast<const ResT*>(res_in) + static_cast<size_t>(t) * H + h);
  for (int j0 = 0; j0 < k; j0 += kSlotBatch) {
    f32x4 v[kSlotBatch];
    float wj[kSlotBatch];
    if constexpr (kF16S) {
      const uint16_t* hv = static_cast<const uint16_t*>(slot_out);
      const int8_t* ev = reinterpret_cast<const int8_t*>(hv + static_cast<size_t>(T) * k * H);
      const int h16 = H >> 4;
      uint2 q[kSlotBatch];
      int ex[kSlotBatch];
#pragma unroll
      for (int u = 0; u < kSlotBatch; ++u)
        if (j0 + u < k) {
          const size_t row = row0 + j0 + u;
          q[u] = *reinterpret_cast<const uint2*>(hv + row * H + h);
          ex[u] = ev[row * h16 + (h >> 4)];
          wj[u] = wt[j0 + u];
        }
#pragma unroll
      for (int u = 0; u < kSlotBatch; ++u)
        if (j0 + u < k) v[u] = f16s_decode(q[u], ex[u]);
    } else {
      const float* so = static_cast<const float*>(slot_out);
#pragma unroll
      for (int u = 0; u < kSlotBatch; ++u)
        if (j0 + u < k) {
          v[u] = *reinterpret_cast<const f32x4*>(so + (row0 + j0 + u) * H + h);
          wj[u] = wt[j0 + u];
        }
    }
#pragma unroll
    for (int u = 0; u < kSlotBatch; ++u)
      if (j0 + u < k) acc += wj[u] * v[u];  // slot order
  }
  if (shared_out) acc += sh;
  store4(y + static_cast<size_t>(t) * H + h, acc);
  if constexpr (!std::is_void_v<ResT>) store4(static_cast<ResT*>(res_out) + static_cast<size_t>(t) * H + h, rv + acc);
}

template <typename OutT, bool kF16S>
hipError_t launch_combine_res(unsigned blocks, const void* slot_out, const float* w, const float* shared_out, int T,
                              int H, int k, OutT* y, const void* res_in, void* res_out, dmoe_dtype res_dt,
                              hipStream_t s) {
  if (!res_out)
    combine_kernel<OutT, kF16S, void><<<blocks, kCombineThreads, 0, s>>>(slot_out, w, shared_out, T, H, k, y,
                                                                          nullptr, nullptr);
  else if (res_dt == DMOE_BF16)
    combine_kernel<OutT, kF16S, bf16_t><<<blocks, kCombineThreads, 0, s>>>(slot_out, w, shared_out, T, H, k, y,
                                                                            res_in, res_out);
  else
    combine_kernel<OutT, kF16S, float><<<blocks, kCombineThreads, 0, s>>>(slot_out, w, shared_out, T, H, k, y,
                                                                           res_in, res_out);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_combine(const void* slot_out, dmoe_slot_format slot_fmt, const float* w,
                          const float* shared_out, dmoe_dtype dt, int T, int H, int k, void* y, hipStream_t s,
                          const void* res_in, void* res_out, dmoe_dtype res_dt) {
  const size_t n = static_cast<size_t>(T) * (H >> 2);
  const unsigned blocks = static_cast<unsigned>((n + kCombineThreads - 1) / kCombineThreads);
  const bool f16s = slot_fmt == DMOE_SLOT_F16S;
  if (dt == DMOE_BF16) {
    bf16_t* yb = static_cast<bf16_t*>(y);
    return f16s ? launch_combine_res<bf16_t, true>(blocks, slot_out, w, shared_out, T, H, k, yb, res_in, res_out,
                                                   res_dt, s)
                : launch_combine_res<bf16_t, false>(blocks, slot_out, w, shared_out, T, H, k, yb, res_in, res_out,
                                                    res_dt, s);
  }
  float* yf = static_cast<float*>(y);
  return f16s ? launch_combine_res<float, true>(blocks, slot_out, w, shared_out, T, H, k, yf, res_in, res_out, res_dt,
                                                s)
              : launch_combine_res<float, false>(blocks, slot_out, w, shared_out, T, H, k, yf, res_in, res_out, res_dt,
                                                 s);
}

}  // namespace dmoe
