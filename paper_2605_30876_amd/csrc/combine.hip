// Weighted combine of the routed expert outputs and the shared expert:
//   y[t][h] = sum_j w[t][j] * slot_out[t][j][h] (+ shared_out[t][h])
// summed in slot order in fp32.  One thread per four consecutive outputs; a
// batch of slot rows is loaded at once (one memory round trip per batch).
// Slot outputs are float32 or scaled half (four fp16 values and the exponent
// byte of their 16-value group per thread and slot, decoded exactly to fp32).
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

template <typename OutT, bool kF16S>
__global__ __launch_bounds__(kCombineThreads) void combine_kernel(const void* __restrict__ slot_out,
                                                      const float* __restrict__ w,
                                                      const float* __restrict__ shared_out, int T,
                                                      int H, int k, OutT* __restrict__ y) {
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
}

}  // namespace

hipError_t launch_combine(const void* slot_out, dmoe_slot_format slot_fmt, const float* w,
                          const float* shared_out, dmoe_dtype dt, int T, int H, int k, void* y, hipStream_t s) {
  const size_t n = static_cast<size_t>(T) * (H >> 2);
  const unsigned blocks = static_cast<unsigned>((n + kCombineThreads - 1) / kCombineThreads);
  const bool f16s = slot_fmt == DMOE_SLOT_F16S;
  if (dt == DMOE_BF16) {
    bf16_t* yb = static_cast<bf16_t*>(y);
    if (f16s)
      combine_kernel<bf16_t, true><<<blocks, kCombineThreads, 0, s>>>(slot_out, w, shared_out, T, H, k, yb);
    else
      combine_kernel<bf16_t, false><<<blocks, kCombineThreads, 0, s>>>(slot_out, w, shared_out, T, H, k, yb);
  } else {
    float* yf = static_cast<float*>(y);
    if (f16s)
      combine_kernel<float, true><<<blocks, kCombineThreads, 0, s>>>(slot_out, w, shared_out, T, H, k, yf);
    else
      combine_kernel<float, false><<<blocks, kCombineThreads, 0, s>>>(slot_out, w, shared_out, T, H, k, yf);
  }
  return hipGetLastError();
}

}  // namespace dmoe
