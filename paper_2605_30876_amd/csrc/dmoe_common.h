// Internal declarations shared by the host validation layer and the gfx950
// kernels of libdmoe.  Not part of the public ABI (see include/dmoe.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "dmoe.h"

namespace dmoe {

// ---------------------------------------------------------------------------
// Element types
// ---------------------------------------------------------------------------
typedef uint16_t bf16_t;  // bfloat16 storage: the upper 16 bits of a binary32
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ float bf16_to_f32(bf16_t v) {
  return __uint_as_float(static_cast<uint32_t>(v) << 16);
}

// Round-to-nearest-even binary32 -> bfloat16 (NaN stays a quiet NaN).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return static_cast<bf16_t>((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<bf16_t>(u >> 16);
}

template <typename T>
__device__ __forceinline__ float load_as_f32(const T* p);
template <>
__device__ __forceinline__ float load_as_f32<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float load_as_f32<bf16_t>(const bf16_t* p) { return bf16_to_f32(*p); }

template <typename T>
__device__ __forceinline__ void store_from_f32(T* p, float v);
template <>
__device__ __forceinline__ void store_from_f32<float>(float* p, float v) { *p = v; }
template <>
__device__ __forceinline__ void store_from_f32<bf16_t>(bf16_t* p, float v) { *p = f32_to_bf16(v); }

// 16-byte load of eight bfloat16 values as an MFMA operand.
__device__ __forceinline__ bf16x8 ld_bf16x8(const bf16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(p));
}

// A non-temporal load (no reuse expected: weights a forward streams once).
// Measured on MI355X, streaming reads over every CU reach ~7.1-7.3 TB/s this
// way against ~5.9-6.2 TB/s with plain loads.
__device__ __forceinline__ bf16x8 ld_bf16x8_stream(const bf16_t* p) {
  return __builtin_bit_cast(bf16x8, __builtin_nontemporal_load(reinterpret_cast<const u16x8*>(p)));
}

__device__ __forceinline__ float silu_f32(float a) { return a / (1.0f + expf(-a)); }

// DMOE_SLOT_F16S: sixteen consecutive outputs share a power-of-two exponent
// e (int8) and each is stored as the fp16 rounding (to nearest even) of
// v * 2^-e.  e puts the largest finite |v| of the sixteen in [2^14, 2^15), so
// nothing overflows and every value within 2^28 of that maximum keeps fp16's
// 11 significant bits; NaN and infinities stay NaN and infinite.  A lane
// holds four of the sixteen (a matrix-core output row of 16 features is
// spread over the four lanes c, c + 16, c + 32, c + 48): f16s_group_max
// combines their maxima, so all 64 lanes of the wave must call it.
__device__ __forceinline__ float f16s_group_max(const f32x4& v) {
  float m = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float a = fabsf(v[i]);
    m = a <= 3.40282347e38f ? fmaxf(m, a) : m;  // finite values only (NaN compares false)
  }
  // lanes i and i ^ 32, then i and i ^ 16: the gfx950 lane-swap
  // instructions (VALU, no LDS round trip) hand each lane the other half's value
  const auto s32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
  m = fmaxf(__uint_as_float(s32[0]), __uint_as_float(s32[1]));
  const auto s16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(m), __float_as_uint(m), false, false);
  return fmaxf(__uint_as_float(s16[0]), __uint_as_float(s16[1]));
}

__device__ __forceinline__ int f16s_exponent(float m) {
  int ex = 0;
  if (m > 0.f) (void)frexpf(m, &ex);  // m = f * 2^ex, f in [0.5, 1)
  return m > 0.f ? min(max(ex - 15, -127), 127) : 0;
}

__device__ __forceinline__ uint2 f16s_encode(const f32x4& v, int e) {
  uint32_t b[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) b[i] = __builtin_bit_cast(uint16_t, static_cast<_Float16>(ldexpf(v[i], -e)));
  return make_uint2(b[0] | (b[1] << 16), b[2] | (b[3] << 16));
}

__device__ __forceinline__ f32x4 f16s_decode(uint2 h, int e) {
  const uint32_t b[4] = {h.x & 0xffffu, h.x >> 16, h.y & 0xffffu, h.y >> 16};
  f32x4 v;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    v[i] = ldexpf(static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(b[i]))), e);
  return v;
}

// Bytes of slot outputs [T][k][H] in format f (DMOE_SLOT_F16S: the fp16
// values, then one exponent byte per sixteen values).
inline size_t slot_out_bytes(long T, long H, long k, dmoe_slot_format f) {
  return f == DMOE_SLOT_F16S ? static_cast<size_t>(T * k * H * 2 + T * k * (H / 16))
                             : static_cast<size_t>(T * k * H * 4);
}

constexpr int kWave = 64;  // CDNA wavefront width

// ---------------------------------------------------------------------------
// Host-side launchers (one per kernel family; arguments already validated)
// ---------------------------------------------------------------------------
hipError_t launch_router(const void* x, const void* w, const float* bias, dmoe_dtype dt, int T,
                         int H, int E, float* logits, float* probs, void* x_chunked,
                         void* workspace, size_t ws_bytes, hipStream_t s);
size_t router_workspace_bytes(int T, int H, int E, dmoe_dtype dt);
// Router logits only, as S partial planes [S][T][E] (summed in slice order by
// the softmax) in *part: the workspace when it is large enough, else S = 1
// and *part = probs.
hipError_t launch_router_partials(const void* x, const void* w, dmoe_dtype dt, int T, int H, int E,
                                  float* probs, void* x_chunked, void* workspace, size_t ws_bytes,
                                  hipStream_t s, float** part, int* S);
hipError_t launch_block_topk(const float* probs, int nb, int bs, int E, int k, float* scores,
                             int32_t* experts, float* w, float* gap, hipStream_t s);
// raw: w holds the selected probabilities themselves, not renormalised
// (the Top-P coreset's input; its final selection overwrites them).
hipError_t launch_token_topk(const float* probs, int T, int E, int k, int32_t* experts, float* w,
                             float* gap, hipStream_t s, bool raw = false);
// Softmax of the router's S partial logit planes and token top-k in one
// launch (E <= 512); probs, weights and selections as the two-step chain.
bool softmax_token_topk_fits(int E);
hipError_t launch_softmax_token_topk(const float* part, int S, const float* bias, int T, int E, int k, float* probs,
                                     float* logits, int32_t* experts, float* w, float* gap, hipStream_t s,
                                     bool raw = false);
hipError_t launch_schedule(const int32_t* experts, int n_groups, int gs, int k, int E,
                           dmoe_schedule sched, hipStream_t s);
hipError_t launch_block_topp(const float* probs, int nb, int bs, int E, int k, float p, int min_c,
                             float* block_scores, int32_t* coreset, int32_t* coreset_size, int32_t* experts,
                             float* w, float* gap, hipStream_t s, bool own_done = false);
bool topp_supported(int bs, int E, int k);

// The whole routing stage: router, selection (blocks of gs tokens when block,
// else per token), combine weights and schedule.  Small forwards run the
// selection and schedule in one workgroup after the router; others chain the
// separate launchers.  Results are identical either way.
struct RouteArgs {
  const void* x;
  const void* w;
  const float* bias;
  int T, H, E, k, gs;
  bool block;
  float* logits;
  float* probs;
  void* x_chunked;
  float* block_scores;
  int32_t* experts;
  float* combine_w;
  float* gap;
  dmoe_schedule sched;
  void* workspace;
  size_t ws_bytes;
  // Alg. 1 with the Top-P coreset (block = false; gs is the block size)
  bool topp = false;
  float top_p = 0.f;
  int min_coreset = 0;
  int32_t* coreset = nullptr;
  int32_t* coreset_size = nullptr;
};
hipError_t launch_route(const RouteArgs& a, dmoe_dtype dt, hipStream_t s);
bool route_fused_fits(int T, int E, int k, int gs, bool block);

// 16-byte chunks: elements of one chunk of the chunk-major activation layout.
inline int chunk_elems(dmoe_dtype dt) { return dt == DMOE_F32 ? 4 : 8; }
inline size_t dtype_bytes(dmoe_dtype dt) { return dt == DMOE_F32 ? 4 : 2; }

hipError_t launch_pack_weights(const void* wg, const void* wu, const void* wd, dmoe_dtype dt, int E,
                               int H, int I, void* w13, void* w2, hipStream_t s);
hipError_t launch_pack_activations(const void* x, dmoe_dtype dt, int T, int H, void* x_chunked,
                                   hipStream_t s);

struct FfnArgs {
  const void* x;     // activations, chunk-major [H/c][T][c]
  const void* xr;    // the same activations row-major [T][H], or nullptr
  const void* w13;   // packed routed gate/up weights
  const void* w2;    // packed routed down weights
  const void* ws13;  // packed shared-expert gate/up (or nullptr)
  const void* ws2;   // packed shared-expert down (or nullptr)
  int T, H, E, I, I_s, k, max_work;
  dmoe_schedule sched;
  void* slot_out;
  dmoe_slot_format slot_fmt;
  float* shared_out;
  void* workspace;  // SwiGLU activations of T*k (+ T) rows, max(I, I_s) wide, storage type
};
hipError_t launch_ffn(const FfnArgs& a, dmoe_dtype dt, hipStream_t s);
// Device address of this device's DMOE_NOALLOC_SCRATCH_BYTES scratch array
// (looked up on the first call per device, then cached).
hipError_t noalloc_scratch(void** ptr);
size_t ffn_workspace_bytes(int T, int I, int I_s, int k, dmoe_dtype dt);
long schedule_max_work(long n_groups, long group_size, long k, long E);
size_t schedule_scratch_ints(long n_groups, long k, long E);

// The whole block-routed layer of one block in three launches (layer.hip):
// router + shared gate/up, routing + routed gate/up, down + combine.
struct LayerArgs {
  const void* x;
  const void* w_router;
  const float* bias;
  const void* w13;
  const void* w2;
  const void* ws13;  // nullptr: no shared expert
  const void* ws2;
  int T, H, E, I, I_s, k;
  float* logits;  // or nullptr
  float* probs;
  void* x_chunked;
  float* block_scores;  // or nullptr
  int32_t* experts;
  float* combine_w;
  float* gap;  // or nullptr
  dmoe_schedule sched;
  void* workspace;  // layer_fused_workspace_bytes
  void* y;
  dmoe_dtype y_dt;
  const void* res_in;  // residual: res_out = bf16(res_in + y), or nullptr
  void* res_out;
};
bool layer_fused_fits(dmoe_dtype dt, int n_blocks, int T, int H, int E, int I, int I_s, int k);
size_t layer_fused_workspace_bytes(int T, int E, int I, int I_s, int k);
hipError_t launch_layer_fused(const LayerArgs& a, hipStream_t s);

// res_out (optional): res_out = round_res_dt(res_in + y) from the fp32 sum.
hipError_t launch_combine(const void* slot_out, dmoe_slot_format slot_fmt, const float* w,
                          const float* shared_out, dmoe_dtype dt, int T, int H, int k, void* y, hipStream_t s,
                          const void* res_in = nullptr, void* res_out = nullptr, dmoe_dtype res_dt = DMOE_BF16);

}  // namespace dmoe
