// Weighted combine of the routed expert outputs and the shared expert:
//   y[t][h] = sum_j w[t][j] * slot_out[t][j][h] (+ shared_out[t][h])
// summed in slot order in fp32.  One thread per four consecutive outputs.
#include "dmoe_common.h"

namespace dmoe {
namespace {

template <typename OutT>
__global__ __launch_bounds__(256) void combine_kernel(const float* __restrict__ slot_out,
                                                      const float* __restrict__ w,
                                                      const float* __restrict__ shared_out, int T,
                                                      int H, int k, OutT* __restrict__ y) {
  const int h4 = H >> 2;
  const size_t idx = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= static_cast<size_t>(T) * h4) return;
  const int t = static_cast<int>(idx / h4);
  const int h = static_cast<int>(idx - static_cast<size_t>(t) * h4) * 4;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  const float* wt = w + static_cast<size_t>(t) * k;
  const float* so = slot_out + static_cast<size_t>(t) * k * H + h;
  for (int j = 0; j < k; ++j) {
    const f32x4 v = *reinterpret_cast<const f32x4*>(so + static_cast<size_t>(j) * H);
    acc += wt[j] * v;
  }
  if (shared_out) acc += *reinterpret_cast<const f32x4*>(shared_out + static_cast<size_t>(t) * H + h);
  OutT* dst = y + static_cast<size_t>(t) * H + h;
#pragma unroll
  for (int i = 0; i < 4; ++i) store_from_f32<OutT>(dst + i, acc[i]);
}

}  // namespace

hipError_t launch_combine(const float* slot_out, const float* w, const float* shared_out,
                          dmoe_dtype dt, int T, int H, int k, void* y, hipStream_t s) {
  const size_t n = static_cast<size_t>(T) * (H >> 2);
  const unsigned blocks = static_cast<unsigned>((n + 255) / 256);
  if (dt == DMOE_BF16)
    combine_kernel<bf16_t><<<blocks, 256, 0, s>>>(slot_out, w, shared_out, T, H, k, static_cast<bf16_t*>(y));
  else
    combine_kernel<float><<<blocks, 256, 0, s>>>(slot_out, w, shared_out, T, H, k, static_cast<float*>(y));
  return hipGetLastError();
}

}  // namespace dmoe
