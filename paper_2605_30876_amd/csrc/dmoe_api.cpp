// C ABI of libdmoe: argument validation on the host, then the kernel
// launchers.  Validation touches no GPU state, so every error path can be
// exercised on a machine without a GPU.
#include <cstdarg>
#include <cstdio>
#include <string>

#include "dmoe_common.h"

namespace {

thread_local std::string g_last_error;

dmoe_status fail(dmoe_status st, const char* fn, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = std::string(fn) + ": " + buf;
  return st;
}

dmoe_status ok() {
  g_last_error.clear();
  return DMOE_OK;
}

dmoe_status hip_status(hipError_t err, const char* fn) {
  if (err == hipSuccess) return ok();
  return fail(DMOE_ERR_HIP, fn, "kernel launch failed: %s", hipGetErrorString(err));
}

bool misaligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; }

bool valid_dtype(dmoe_dtype dt) { return dt == DMOE_F32 || dt == DMOE_BF16; }
bool valid_slot_format(dmoe_slot_format f) { return f == DMOE_SLOT_F32 || f == DMOE_SLOT_F16S; }

constexpr int kMaxE = 4096;
constexpr int kMaxScheduleE = 512;
constexpr int kMaxK = 64;
constexpr long kIntLimit = 0x7fffffffL;

// Name of the entry point in error messages.
#define DMOE_FN __func__
#define REQUIRE(cond, ...)                                  \
  do {                                                      \
    if (!(cond)) return fail(DMOE_ERR_INVALID_ARG, DMOE_FN, __VA_ARGS__); \
  } while (0)
#define SUPPORT(cond, ...)                                  \
  do {                                                      \
    if (!(cond)) return fail(DMOE_ERR_UNSUPPORTED, DMOE_FN, __VA_ARGS__); \
  } while (0)
#define ALIGNED(p) REQUIRE(!misaligned(p), #p " is not 16-byte aligned")

}  // namespace

extern "C" {

const char* dmoe_last_error(void) { return g_last_error.c_str(); }

const char* dmoe_version(void) { return "0.1.0"; }

size_t dmoe_router_workspace_size(int T, int H, int E, dmoe_dtype dt) {
  if (T < 1 || H < 1 || E < 1 || E > kMaxE || !valid_dtype(dt)) return 0;
  return dmoe::router_workspace_bytes(T, H, E, dt);
}

dmoe_status dmoe_router_logits(const void* x, const void* w_router, const float* bias,
                               dmoe_dtype dt, int T, int H, int E, float* logits, float* probs,
                               void* x_chunked, void* workspace, size_t ws_bytes, void* stream) {
  REQUIRE(x && w_router && probs, "x, w_router and probs must not be NULL");
  REQUIRE(valid_dtype(dt), "unknown dtype %d", static_cast<int>(dt));
  REQUIRE(T >= 1 && H >= 1, "T=%d and H=%d must be >= 1", T, H);
  REQUIRE(E >= 1 && E <= kMaxE, "E=%d must be in [1, %d]", E, kMaxE);
  REQUIRE(static_cast<long>(T) * E <= kIntLimit && static_cast<long>(T) * H <= kIntLimit,
          "T*E and T*H must fit in int32");
  ALIGNED(x);
  ALIGNED(w_router);
  ALIGNED(bias);
  ALIGNED(logits);
  ALIGNED(probs);
  ALIGNED(workspace);
  ALIGNED(x_chunked);
  if (x_chunked) {
    REQUIRE(H % dmoe::chunk_elems(dt) == 0, "x_chunked needs H %% %d == 0 (H=%d)", dmoe::chunk_elems(dt), H);
  }
  if (dt == DMOE_BF16) {
    SUPPORT(H % 128 == 0, "bf16 router needs H %% 128 == 0 (H=%d)", H);
  }
  return hip_status(dmoe::launch_router(x, w_router, bias, dt, T, H, E, logits, probs, x_chunked,
                                        workspace, workspace ? ws_bytes : 0,
                                        static_cast<hipStream_t>(stream)),
                    __func__);
}

dmoe_status dmoe_block_aggregate_topk(const float* probs, int n_blocks, int block_size, int E,
                                      int k, float* block_scores, int32_t* block_experts,
                                      float* combine_w, float* gap, void* stream) {
  REQUIRE(probs && block_experts && combine_w, "probs, block_experts and combine_w must not be NULL");
  REQUIRE(n_blocks >= 1, "n_blocks=%d must be >= 1", n_blocks);
  REQUIRE(block_size >= 1 && block_size <= 4096, "block_size=%d must be in [1, 4096]", block_size);
  REQUIRE(E >= 1 && E <= kMaxE, "E=%d must be in [1, %d]", E, kMaxE);
  REQUIRE(k >= 1 && k <= E && k <= kMaxK, "k=%d must be in [1, min(E, %d)]", k, kMaxK);
  REQUIRE(static_cast<long>(n_blocks) * block_size * E <= kIntLimit, "T*E must fit in int32");
  ALIGNED(probs);
  ALIGNED(block_scores);
  ALIGNED(block_experts);
  ALIGNED(combine_w);
  ALIGNED(gap);
  return hip_status(dmoe::launch_block_topk(probs, n_blocks, block_size, E, k, block_scores,
                                            block_experts, combine_w, gap,
                                            static_cast<hipStream_t>(stream)),
                    __func__);
}

dmoe_status dmoe_token_topk(const float* probs, int T, int E, int k, int32_t* token_experts,
                            float* combine_w, float* gap, void* stream) {
  REQUIRE(probs && token_experts && combine_w, "probs, token_experts and combine_w must not be NULL");
  REQUIRE(T >= 1, "T=%d must be >= 1", T);
  REQUIRE(E >= 1 && E <= kMaxE, "E=%d must be in [1, %d]", E, kMaxE);
  REQUIRE(k >= 1 && k <= E && k <= kMaxK, "k=%d must be in [1, min(E, %d)]", k, kMaxK);
  REQUIRE(static_cast<long>(T) * E <= kIntLimit, "T*E must fit in int32");
  ALIGNED(probs);
  ALIGNED(token_experts);
  ALIGNED(combine_w);
  ALIGNED(gap);
  return hip_status(dmoe::launch_token_topk(probs, T, E, k, token_experts, combine_w, gap,
                                            static_cast<hipStream_t>(stream)),
                    __func__);
}

dmoe_status dmoe_block_topp_route(const float* probs, int n_blocks, int block_size, int E, int k, float p,
                                  int min_coreset, float* block_scores, int32_t* coreset, int32_t* coreset_size,
                                  int32_t* token_experts, float* combine_w, float* gap, void* stream) {
  REQUIRE(probs && coreset && coreset_size && token_experts && combine_w,
          "probs, coreset, coreset_size, token_experts and combine_w must not be NULL");
  REQUIRE(n_blocks >= 1, "n_blocks=%d must be >= 1", n_blocks);
  REQUIRE(block_size >= 1 && block_size <= 4096, "block_size=%d must be in [1, 4096]", block_size);
  REQUIRE(E >= 1 && E <= kMaxE, "E=%d must be in [1, %d]", E, kMaxE);
  REQUIRE(k >= 1 && k <= E && k <= kMaxK, "k=%d must be in [1, min(E, %d)]", k, kMaxK);
  REQUIRE(min_coreset >= k && min_coreset <= E, "min_coreset=%d must be in [k, E]", min_coreset);
  REQUIRE(p > 0.f && p <= 1.f, "p=%g must be in (0, 1]", static_cast<double>(p));
  REQUIRE(static_cast<long>(n_blocks) * block_size * E <= kIntLimit, "T*E must fit in int32");
  ALIGNED(probs);
  ALIGNED(block_scores);
  ALIGNED(coreset);
  ALIGNED(coreset_size);
  ALIGNED(token_experts);
  ALIGNED(combine_w);
  ALIGNED(gap);
  SUPPORT(E <= 1024, "the Top-P coreset supports E <= 1024 (E=%d)", E);
  SUPPORT(dmoe::topp_supported(block_size, E, k), "the Top-P kernels do not support block_size=%d, E=%d, k=%d",
          block_size, E, k);
  return hip_status(dmoe::launch_block_topp(probs, n_blocks, block_size, E, k, p, min_coreset, block_scores,
                                            coreset, coreset_size, token_experts, combine_w, gap,
                                            static_cast<hipStream_t>(stream)),
                    __func__);
}

dmoe_status dmoe_build_expert_schedule(const int32_t* experts, int n_groups, int group_size, int k,
                                       int E, dmoe_schedule sched, void* stream) {
  REQUIRE(experts, "experts must not be NULL");
  REQUIRE(sched.n_unique && sched.unique && sched.offsets && sched.row_token && sched.row_slot && sched.n_work &&
              sched.work,
          "every schedule array must be set");
  REQUIRE(n_groups >= 1 && group_size >= 1, "n_groups=%d and group_size=%d must be >= 1", n_groups,
          group_size);
  REQUIRE(E >= 1, "E=%d must be >= 1", E);
  REQUIRE(k >= 1 && k <= E && k <= kMaxK, "k=%d must be in [1, min(E, %d)]", k, kMaxK);
  REQUIRE(static_cast<long>(n_groups) * group_size * k < kIntLimit, "n_groups*group_size*k must fit in int32");
  SUPPORT(E <= kMaxScheduleE, "the schedule supports E <= %d (E=%d)", kMaxScheduleE, E);
  ALIGNED(experts);
  ALIGNED(sched.n_unique);
  ALIGNED(sched.unique);
  ALIGNED(sched.offsets);
  ALIGNED(sched.scratch);
  ALIGNED(sched.row_token);
  ALIGNED(sched.row_slot);
  ALIGNED(sched.n_work);
  ALIGNED(sched.work);
  return hip_status(dmoe::launch_schedule(experts, n_groups, group_size, k, E, sched,
                                          static_cast<hipStream_t>(stream)),
                    __func__);
}

dmoe_status dmoe_route_block(const void* x, const void* w_router, const float* bias, dmoe_dtype dt,
                             int n_blocks, int block_size, int H, int E, int k, float* logits,
                             float* probs, void* x_chunked, float* block_scores, int32_t* block_experts,
                             float* combine_w, float* gap, dmoe_schedule sched, void* workspace,
                             size_t ws_bytes, void* stream) {
  REQUIRE(x && w_router && probs && block_experts && combine_w,
          "x, w_router, probs, block_experts and combine_w must not be NULL");
  REQUIRE(sched.n_unique && sched.unique && sched.offsets && sched.row_token && sched.row_slot && sched.n_work &&
              sched.work,
          "every schedule array must be set");
  REQUIRE(valid_dtype(dt), "unknown dtype %d", static_cast<int>(dt));
  REQUIRE(n_blocks >= 1, "n_blocks=%d must be >= 1", n_blocks);
  REQUIRE(block_size >= 1 && block_size <= 4096, "block_size=%d must be in [1, 4096]", block_size);
  REQUIRE(H >= 1, "H=%d must be >= 1", H);
  REQUIRE(E >= 1 && E <= kMaxE, "E=%d must be in [1, %d]", E, kMaxE);
  REQUIRE(k >= 1 && k <= E && k <= kMaxK, "k=%d must be in [1, min(E, %d)]", k, kMaxK);
  const long T = static_cast<long>(n_blocks) * block_size;
  REQUIRE(T * E <= kIntLimit && T * H <= kIntLimit && T * k < kIntLimit, "T*E, T*H and T*k must fit in int32");
  ALIGNED(x);
  ALIGNED(w_router);
  ALIGNED(bias);
  ALIGNED(logits);
  ALIGNED(probs);
  ALIGNED(x_chunked);
  ALIGNED(block_scores);
  ALIGNED(block_experts);
  ALIGNED(combine_w);
  ALIGNED(gap);
  ALIGNED(workspace);
  ALIGNED(sched.n_unique);
  ALIGNED(sched.unique);
  ALIGNED(sched.offsets);
  ALIGNED(sched.scratch);
  ALIGNED(sched.row_token);
  ALIGNED(sched.row_slot);
  ALIGNED(sched.n_work);
  ALIGNED(sched.work);
  if (x_chunked) {
    REQUIRE(H % dmoe::chunk_elems(dt) == 0, "x_chunked needs H %% %d == 0 (H=%d)", dmoe::chunk_elems(dt), H);
  }
  if (dt == DMOE_BF16) {
    SUPPORT(H % 128 == 0, "bf16 router needs H %% 128 == 0 (H=%d)", H);
  }
  SUPPORT(E <= kMaxScheduleE, "the schedule supports E <= %d (E=%d)", kMaxScheduleE, E);
  dmoe::RouteArgs a{x, w_router, bias, static_cast<int>(T), H, E, k, block_size, true, logits, probs,
                    x_chunked, block_scores, block_experts, combine_w, gap, sched, workspace,
                    workspace ? ws_bytes : 0};
  return hip_status(dmoe::launch_route(a, dt, static_cast<hipStream_t>(stream)), __func__);
}

dmoe_status dmoe_route_token(const void* x, const void* w_router, const float* bias, dmoe_dtype dt,
                             int T, int H, int E, int k, float* logits, float* probs, void* x_chunked,
                             int32_t* token_experts, float* combine_w, float* gap, dmoe_schedule sched,
                             void* workspace, size_t ws_bytes, void* stream) {
  REQUIRE(x && w_router && probs && token_experts && combine_w,
          "x, w_router, probs, token_experts and combine_w must not be NULL");
  REQUIRE(sched.n_unique && sched.unique && sched.offsets && sched.row_token && sched.row_slot && sched.n_work &&
              sched.work,
          "every schedule array must be set");
  REQUIRE(valid_dtype(dt), "unknown dtype %d", static_cast<int>(dt));
  REQUIRE(T >= 1 && H >= 1, "T=%d and H=%d must be >= 1", T, H);
  REQUIRE(E >= 1 && E <= kMaxE, "E=%d must be in [1, %d]", E, kMaxE);
  REQUIRE(k >= 1 && k <= E && k <= kMaxK, "k=%d must be in [1, min(E, %d)]", k, kMaxK);
  REQUIRE(static_cast<long>(T) * E <= kIntLimit && static_cast<long>(T) * H <= kIntLimit &&
              static_cast<long>(T) * k < kIntLimit,
          "T*E, T*H and T*k must fit in int32");
  ALIGNED(x);
  ALIGNED(w_router);
  ALIGNED(bias);
  ALIGNED(logits);
  ALIGNED(probs);
  ALIGNED(x_chunked);
  ALIGNED(token_experts);
  ALIGNED(combine_w);
  ALIGNED(gap);
  ALIGNED(workspace);
  ALIGNED(sched.n_unique);
  ALIGNED(sched.unique);
  ALIGNED(sched.offsets);
  ALIGNED(sched.scratch);
  ALIGNED(sched.row_token);
  ALIGNED(sched.row_slot);
  ALIGNED(sched.n_work);
  ALIGNED(sched.work);
  if (x_chunked) {
    REQUIRE(H % dmoe::chunk_elems(dt) == 0, "x_chunked needs H %% %d == 0 (H=%d)", dmoe::chunk_elems(dt), H);
  }
  if (dt == DMOE_BF16) {
    SUPPORT(H % 128 == 0, "bf16 router needs H %% 128 == 0 (H=%d)", H);
  }
  SUPPORT(E <= kMaxScheduleE, "the schedule supports E <= %d (E=%d)", kMaxScheduleE, E);
  dmoe::RouteArgs a{x, w_router, bias, T, H, E, k, 1, false, logits, probs, x_chunked, nullptr, token_experts,
                    combine_w, gap, sched, workspace, workspace ? ws_bytes : 0};
  return hip_status(dmoe::launch_route(a, dt, static_cast<hipStream_t>(stream)), __func__);
}

dmoe_status dmoe_route_topp(const void* x, const void* w_router, const float* bias, dmoe_dtype dt, int n_blocks,
                            int block_size, int H, int E, int k, float p, int min_coreset, float* logits,
                            float* probs, void* x_chunked, float* block_scores, int32_t* coreset,
                            int32_t* coreset_size, int32_t* token_experts, float* combine_w, float* gap,
                            dmoe_schedule sched, void* workspace, size_t ws_bytes, void* stream) {
  REQUIRE(x && w_router && probs && coreset && coreset_size && token_experts && combine_w,
          "x, w_router, probs, coreset, coreset_size, token_experts and combine_w must not be NULL");
  REQUIRE(sched.n_unique && sched.unique && sched.offsets && sched.row_token && sched.row_slot && sched.n_work &&
              sched.work,
          "every schedule array must be set");
  REQUIRE(valid_dtype(dt), "unknown dtype %d", static_cast<int>(dt));
  REQUIRE(n_blocks >= 1, "n_blocks=%d must be >= 1", n_blocks);
  REQUIRE(block_size >= 1 && block_size <= 4096, "block_size=%d must be in [1, 4096]", block_size);
  REQUIRE(H >= 1, "H=%d must be >= 1", H);
  REQUIRE(E >= 1 && E <= kMaxE, "E=%d must be in [1, %d]", E, kMaxE);
  REQUIRE(k >= 1 && k <= E && k <= kMaxK, "k=%d must be in [1, min(E, %d)]", k, kMaxK);
  REQUIRE(min_coreset >= k && min_coreset <= E, "min_coreset=%d must be in [k, E]", min_coreset);
  REQUIRE(p > 0.f && p <= 1.f, "p=%g must be in (0, 1]", static_cast<double>(p));
  const long T = static_cast<long>(n_blocks) * block_size;
  REQUIRE(T * E <= kIntLimit && T * H <= kIntLimit && T * k < kIntLimit, "T*E, T*H and T*k must fit in int32");
  ALIGNED(x);
  ALIGNED(w_router);
  ALIGNED(bias);
  ALIGNED(logits);
  ALIGNED(probs);
  ALIGNED(x_chunked);
  ALIGNED(block_scores);
  ALIGNED(coreset);
  ALIGNED(coreset_size);
  ALIGNED(token_experts);
  ALIGNED(combine_w);
  ALIGNED(gap);
  ALIGNED(workspace);
  ALIGNED(sched.n_unique);
  ALIGNED(sched.unique);
  ALIGNED(sched.offsets);
  ALIGNED(sched.scratch);
  ALIGNED(sched.row_token);
  ALIGNED(sched.row_slot);
  ALIGNED(sched.n_work);
  ALIGNED(sched.work);
  if (x_chunked) {
    REQUIRE(H % dmoe::chunk_elems(dt) == 0, "x_chunked needs H %% %d == 0 (H=%d)", dmoe::chunk_elems(dt), H);
  }
  if (dt == DMOE_BF16) {
    SUPPORT(H % 128 == 0, "bf16 router needs H %% 128 == 0 (H=%d)", H);
  }
  SUPPORT(E <= kMaxScheduleE, "the schedule supports E <= %d (E=%d)", kMaxScheduleE, E);
  SUPPORT(dmoe::topp_supported(block_size, E, k), "the Top-P kernels do not support block_size=%d, E=%d, k=%d",
          block_size, E, k);
  dmoe::RouteArgs a{x, w_router, bias, static_cast<int>(T), H, E, k, block_size, false, logits, probs,
                    x_chunked, block_scores, token_experts, combine_w, gap, sched, workspace,
                    workspace ? ws_bytes : 0};
  a.topp = true;
  a.top_p = p;
  a.min_coreset = min_coreset;
  a.coreset = coreset;
  a.coreset_size = coreset_size;
  return hip_status(dmoe::launch_route(a, dt, static_cast<hipStream_t>(stream)), __func__);
}

dmoe_status dmoe_pack_activations(const void* x, dmoe_dtype dt, int T, int H, void* x_chunked,
                                  void* stream) {
  REQUIRE(x && x_chunked, "x and x_chunked must not be NULL");
  REQUIRE(valid_dtype(dt), "unknown dtype %d", static_cast<int>(dt));
  REQUIRE(T >= 1 && H >= 1, "T=%d and H=%d must be >= 1", T, H);
  REQUIRE(H % dmoe::chunk_elems(dt) == 0, "H=%d must be a multiple of %d", H, dmoe::chunk_elems(dt));
  REQUIRE(static_cast<long>(T) * H <= kIntLimit, "T*H must fit in int32");
  REQUIRE(x != x_chunked, "x and x_chunked must not alias");
  ALIGNED(x);
  ALIGNED(x_chunked);
  return hip_status(dmoe::launch_pack_activations(x, dt, T, H, x_chunked, static_cast<hipStream_t>(stream)),
                    __func__);
}

dmoe_status dmoe_pack_expert_weights(const void* w_gate, const void* w_up, const void* w_down,
                                     dmoe_dtype dt, int n_experts, int H, int I, void* w13, void* w2,
                                     void* stream) {
  REQUIRE(w_gate && w_up && w_down && w13 && w2, "no pointer may be NULL");
  REQUIRE(valid_dtype(dt), "unknown dtype %d", static_cast<int>(dt));
  REQUIRE(n_experts >= 1 && H >= 1 && I >= 1, "n_experts=%d, H=%d and I=%d must be >= 1", n_experts, H, I);
  REQUIRE(w13 != w_gate && w13 != w_up && w13 != w_down && w2 != w_gate && w2 != w_up && w2 != w_down &&
              w13 != w2,
          "outputs must not alias the inputs or each other");
  ALIGNED(w_gate);
  ALIGNED(w_up);
  ALIGNED(w_down);
  ALIGNED(w13);
  ALIGNED(w2);
  if (dt == DMOE_BF16) {
    SUPPORT(H % 128 == 0 && I % 128 == 0, "bf16 experts need H and I to be multiples of 128 (H=%d, I=%d)",
            H, I);
  }
  return hip_status(dmoe::launch_pack_weights(w_gate, w_up, w_down, dt, n_experts, H, I, w13, w2,
                                              static_cast<hipStream_t>(stream)),
                    __func__);
}

int dmoe_schedule_max_work(int n_groups, int group_size, int k, int E) {
  if (n_groups < 1 || group_size < 1 || k < 1 || E < 1 || k > E) return 0;
  const long n = dmoe::schedule_max_work(n_groups, group_size, k, E);
  return n <= kIntLimit ? static_cast<int>(n) : 0;
}

size_t dmoe_schedule_scratch_ints(int n_groups, int k, int E) {
  if (n_groups < 1 || k < 1 || E < 1) return 0;
  return dmoe::schedule_scratch_ints(n_groups, k, E);
}

size_t dmoe_ffn_workspace_size(int T, int I, int I_s, int k, dmoe_dtype dt) {
  if (T < 1 || I < 1 || I_s < 0 || k < 1 || !valid_dtype(dt)) return 0;
  return dmoe::ffn_workspace_bytes(T, I, I_s, k, dt);
}

}  // extern "C"

namespace {

// dmoe_expert_ffn and dmoe_expert_ffn_noalloc: every argument is validated on
// the host first; then (noalloc) the device scratch replaces the workspace.
dmoe_status expert_ffn(const char* fn, const void* x_chunked, const void* x, const void* w13, const void* w2,
                       const void* ws13, const void* ws2, dmoe_dtype dt, int T, int H, int E, int I, int I_s, int k,
                       int max_work, dmoe_schedule sched, void* slot_out, dmoe_slot_format slot_fmt,
                       float* shared_out, void* workspace, size_t ws_bytes, void* stream, bool noalloc) {
#undef DMOE_FN
#define DMOE_FN fn  // messages name the entry point
  REQUIRE(x_chunked && w13 && w2 && slot_out && (workspace || noalloc),
          "x_chunked, w13, w2, slot_out and workspace must not be NULL");
  REQUIRE(sched.n_unique && sched.unique && sched.offsets && sched.row_token && sched.row_slot && sched.n_work &&
              sched.work,
          "every schedule array must be set");
  REQUIRE(valid_dtype(dt), "unknown dtype %d", static_cast<int>(dt));
  REQUIRE(valid_slot_format(slot_fmt), "unknown slot format %d", static_cast<int>(slot_fmt));
  REQUIRE(T >= 1 && H >= 1 && I >= 1 && I_s >= 0, "T=%d, H=%d, I=%d must be >= 1 and I_s=%d >= 0",
          T, H, I, I_s);
  REQUIRE(E >= 1, "E=%d must be >= 1", E);
  REQUIRE(k >= 1 && k <= E && k <= kMaxK, "k=%d must be in [1, min(E, %d)]", k, kMaxK);
  REQUIRE(max_work >= 1 && static_cast<long>(max_work) <= static_cast<long>(T) * k,
          "max_work=%d must be in [1, T*k]", max_work);
  REQUIRE(H % dmoe::chunk_elems(dt) == 0, "H=%d must be a multiple of %d", H, dmoe::chunk_elems(dt));
  const bool shared = I_s > 0;
  REQUIRE(shared == (ws13 != nullptr) && shared == (ws2 != nullptr) && shared == (shared_out != nullptr),
          "ws13, ws2 and shared_out must all be set iff I_s > 0");
  const long rows = static_cast<long>(T) * k + (shared ? T : 0);
  REQUIRE(rows < kIntLimit && rows * (I > I_s ? I : I_s) <= kIntLimit && static_cast<long>(T) * H <= kIntLimit &&
              static_cast<long>(T) * k * H <= kIntLimit * 4L,
          "T*k*H, T*H or the SwiGLU buffer is too large");
  const size_t need = dmoe::ffn_workspace_bytes(T, I, I_s, k, dt);
  if (noalloc) {
    REQUIRE(need <= DMOE_NOALLOC_SCRATCH_BYTES,
            "the SwiGLU activations need %zu bytes, more than the %zu-byte device scratch of this entry point "
            "(call dmoe_expert_ffn with a workspace)",
            need, static_cast<size_t>(DMOE_NOALLOC_SCRATCH_BYTES));
  } else {
    REQUIRE(ws_bytes >= need, "workspace of %zu bytes is smaller than the %zu bytes needed", ws_bytes, need);
  }
  ALIGNED(x_chunked);
  ALIGNED(x);
  ALIGNED(w13);
  ALIGNED(w2);
  ALIGNED(sched.n_work);
  ALIGNED(sched.work);
  ALIGNED(sched.row_token);
  ALIGNED(sched.row_slot);
  ALIGNED(ws13);
  ALIGNED(ws2);
  ALIGNED(slot_out);
  ALIGNED(shared_out);
  ALIGNED(workspace);
  SUPPORT(E <= kMaxScheduleE, "E <= %d is supported (E=%d)", kMaxScheduleE, E);
  if (dt == DMOE_BF16) {
    SUPPORT(H % 128 == 0 && I % 128 == 0 && I_s % 128 == 0,
            "bf16 experts need H, I and I_s to be multiples of 128 (H=%d, I=%d, I_s=%d)", H, I, I_s);
  }
  SUPPORT(slot_fmt == DMOE_SLOT_F32 || dt == DMOE_BF16, "scaled-half slot outputs need DMOE_BF16 experts");
  if (noalloc) {
    const hipError_t err = dmoe::noalloc_scratch(&workspace);
    if (err != hipSuccess) return fail(DMOE_ERR_HIP, fn, "device scratch lookup failed: %s", hipGetErrorString(err));
  }
  dmoe::FfnArgs a{x_chunked, x, w13, w2, ws13, ws2, T, H, E, I, I_s, k, max_work,
                  sched, slot_out, slot_fmt, shared_out, workspace};
  return hip_status(dmoe::launch_ffn(a, dt, static_cast<hipStream_t>(stream)), fn);
}
#undef DMOE_FN
#define DMOE_FN __func__

}  // namespace

extern "C" {

dmoe_status dmoe_expert_ffn(const void* x_chunked, const void* x, const void* w13, const void* w2,
                            const void* ws13, const void* ws2, dmoe_dtype dt, int T, int H, int E, int I,
                            int I_s, int k, int max_work, dmoe_schedule sched, void* slot_out,
                            dmoe_slot_format slot_fmt, float* shared_out, void* workspace, size_t ws_bytes,
                            void* stream) {
  return expert_ffn(__func__, x_chunked, x, w13, w2, ws13, ws2, dt, T, H, E, I, I_s, k, max_work, sched, slot_out,
                    slot_fmt, shared_out, workspace, ws_bytes, stream, false);
}

dmoe_status dmoe_expert_ffn_noalloc(const void* x_chunked, const void* x, const void* w13, const void* w2,
                                    const void* ws13, const void* ws2, dmoe_dtype dt, int T, int H, int E, int I,
                                    int I_s, int k, int max_work, dmoe_schedule sched, void* slot_out,
                                    dmoe_slot_format slot_fmt, float* shared_out, void* stream) {
  return expert_ffn(__func__, x_chunked, x, w13, w2, ws13, ws2, dt, T, H, E, I, I_s, k, max_work, sched, slot_out,
                    slot_fmt, shared_out, nullptr, 0, stream, true);
}

size_t dmoe_shared_ffn_workspace_size(int T, int I_s, dmoe_dtype dt) {
  if (T < 1 || I_s < 1 || !valid_dtype(dt)) return 0;
  return dmoe::ffn_workspace_bytes(T, 0, I_s, 0, dt);
}

dmoe_status dmoe_shared_expert_ffn(const void* x_chunked, const void* ws13, const void* ws2, dmoe_dtype dt, int T,
                                   int H, int I_s, float* shared_out, void* workspace, size_t ws_bytes,
                                   void* stream) {
  REQUIRE(x_chunked && ws13 && ws2 && shared_out && workspace,
          "x_chunked, ws13, ws2, shared_out and workspace must not be NULL");
  REQUIRE(valid_dtype(dt), "unknown dtype %d", static_cast<int>(dt));
  REQUIRE(T >= 1 && H >= 1 && I_s >= 1, "T=%d, H=%d and I_s=%d must be >= 1", T, H, I_s);
  REQUIRE(H % dmoe::chunk_elems(dt) == 0, "H=%d must be a multiple of %d", H, dmoe::chunk_elems(dt));
  REQUIRE(static_cast<long>(T) * I_s <= kIntLimit && static_cast<long>(T) * H <= kIntLimit,
          "T*H or the SwiGLU buffer is too large");
  const size_t need = dmoe::ffn_workspace_bytes(T, 0, I_s, 0, dt);
  REQUIRE(ws_bytes >= need, "workspace of %zu bytes is smaller than the %zu bytes needed", ws_bytes, need);
  ALIGNED(x_chunked);
  ALIGNED(ws13);
  ALIGNED(ws2);
  ALIGNED(shared_out);
  ALIGNED(workspace);
  if (dt == DMOE_BF16) {
    SUPPORT(H % 128 == 0 && I_s % 128 == 0,
            "bf16 experts need H and I_s to be multiples of 128 (H=%d, I_s=%d)", H, I_s);
  }
  const dmoe_schedule none{};
  dmoe::FfnArgs a{x_chunked, nullptr, nullptr, nullptr, ws13, ws2, T, H, 1, 0, I_s, 0, 0, none, nullptr,
                  DMOE_SLOT_F32, shared_out, workspace};
  return hip_status(dmoe::launch_ffn(a, dt, static_cast<hipStream_t>(stream)), __func__);
}

size_t dmoe_slot_out_bytes(int T, int H, int k, dmoe_slot_format f) {
  if (T < 1 || H < 1 || k < 1 || k > kMaxK || !valid_slot_format(f) || (f == DMOE_SLOT_F16S && H % 16)) return 0;
  return dmoe::slot_out_bytes(T, H, k, f);
}

dmoe_status dmoe_combine(const void* slot_out, dmoe_slot_format slot_fmt, const float* combine_w,
                         const float* shared_out, dmoe_dtype dt, int T, int H, int k, void* y, void* stream) {
  REQUIRE(slot_out && combine_w && y, "slot_out, combine_w and y must not be NULL");
  REQUIRE(valid_dtype(dt), "unknown dtype %d", static_cast<int>(dt));
  REQUIRE(valid_slot_format(slot_fmt), "unknown slot format %d", static_cast<int>(slot_fmt));
  REQUIRE(T >= 1 && H >= 1, "T=%d and H=%d must be >= 1", T, H);
  REQUIRE(H % (slot_fmt == DMOE_SLOT_F16S ? 16 : 4) == 0, "H=%d must be a multiple of %d", H,
          slot_fmt == DMOE_SLOT_F16S ? 16 : 4);
  REQUIRE(k >= 1 && k <= kMaxK, "k=%d must be in [1, %d]", k, kMaxK);
  ALIGNED(slot_out);
  ALIGNED(combine_w);
  ALIGNED(shared_out);
  ALIGNED(y);
  return hip_status(dmoe::launch_combine(slot_out, slot_fmt, combine_w, shared_out, dt, T, H, k, y,
                                         static_cast<hipStream_t>(stream)),
                    __func__);
}

namespace {

size_t align256(size_t n) { return (n + 255) & ~static_cast<size_t>(255); }

// Workspace of the layer: the chained path's router partials and FFN
// activations, or the three-kernel path's logits and weighted activations.
size_t layer_workspace_bytes(int n_blocks, int bs, int H, int E, int I, int I_s, int k, dmoe_dtype dt) {
  const int T = n_blocks * bs;
  const size_t chain = align256(dmoe::router_workspace_bytes(T, H, E, dt)) + dmoe::ffn_workspace_bytes(T, I, I_s, k, dt);
  const size_t fused = dmoe::layer_fused_fits(dt, n_blocks, T, H, E, I, I_s, k)
                           ? dmoe::layer_fused_workspace_bytes(T, E, I, I_s, k)
                           : 0;
  return chain > fused ? chain : fused;
}

}  // namespace

size_t dmoe_moe_forward_workspace_size(int n_blocks, int block_size, int H, int E, int I, int I_s, int k,
                                       dmoe_dtype dt) {
  if (n_blocks < 1 || block_size < 1 || H < 1 || E < 1 || E > kMaxScheduleE || I < 1 || I_s < 0 || k < 1 || k > E ||
      !valid_dtype(dt))
    return 0;
  return layer_workspace_bytes(n_blocks, block_size, H, E, I, I_s, k, dt);
}

int dmoe_moe_forward_fused(dmoe_dtype dt, int n_blocks, int block_size, int H, int E, int I, int I_s, int k,
                           dmoe_routing routing) {
  if (routing != DMOE_ROUTE_BLOCK || !valid_dtype(dt) || n_blocks < 1 || block_size < 1 || block_size > 4096 ||
      H < 1 || H % 4 || I < 1 || I_s < 0 || E < 1 || E > kMaxE || k < 1 || k > E || k > kMaxK)
    return 0;
  return dmoe::layer_fused_fits(dt, n_blocks, n_blocks * block_size, H, E, I, I_s, k) ? 1 : 0;
}

dmoe_status dmoe_moe_forward(const void* x, const void* w_router, const float* bias, const void* w13,
                             const void* w2, const void* ws13, const void* ws2, dmoe_dtype dt, int n_blocks,
                             int block_size, int H, int E, int I, int I_s, int k, dmoe_routing routing, float top_p,
                             int min_coreset, const dmoe_layer_buffers* buf, void* y, dmoe_dtype y_dt,
                             void* stream) {
  // Everything the chained entry points check is checked here first, so a
  // bad argument enqueues nothing.
  REQUIRE(buf, "buf must not be NULL");
  REQUIRE(x && w_router && w13 && w2 && y && buf->probs && buf->x_chunked && buf->experts && buf->combine_w &&
              buf->slot_out && buf->workspace,
          "x, w_router, w13, w2, y and buf's probs, x_chunked, experts, combine_w, slot_out and workspace must "
          "not be NULL");
  const dmoe_schedule& sched = buf->sched;
  REQUIRE(sched.n_unique && sched.unique && sched.offsets && sched.row_token && sched.row_slot && sched.n_work &&
              sched.work,
          "every schedule array must be set");
  REQUIRE(valid_dtype(dt) && valid_dtype(y_dt), "unknown dtype %d / %d", static_cast<int>(dt), static_cast<int>(y_dt));
  REQUIRE(valid_slot_format(buf->slot_fmt), "unknown slot format %d", static_cast<int>(buf->slot_fmt));
  REQUIRE(routing == DMOE_ROUTE_BLOCK || routing == DMOE_ROUTE_TOKEN || routing == DMOE_ROUTE_TOPP,
          "unknown routing %d", static_cast<int>(routing));
  REQUIRE(n_blocks >= 1, "n_blocks=%d must be >= 1", n_blocks);
  REQUIRE(block_size >= 1 && block_size <= 4096, "block_size=%d must be in [1, 4096]", block_size);
  REQUIRE(H >= 1 && I >= 1 && I_s >= 0, "H=%d, I=%d must be >= 1 and I_s=%d >= 0", H, I, I_s);
  REQUIRE(E >= 1 && E <= kMaxE, "E=%d must be in [1, %d]", E, kMaxE);
  REQUIRE(k >= 1 && k <= E && k <= kMaxK, "k=%d must be in [1, min(E, %d)]", k, kMaxK);
  const long T = static_cast<long>(n_blocks) * block_size;
  REQUIRE(T * E <= kIntLimit && T * H <= kIntLimit && T * k < kIntLimit, "T*E, T*H and T*k must fit in int32");
  const bool shared = I_s > 0;
  REQUIRE(shared == (ws13 != nullptr) && shared == (ws2 != nullptr) && shared == (buf->shared_out != nullptr),
          "ws13, ws2 and shared_out must all be set iff I_s > 0");
  const long rows = T * k + (shared ? T : 0);
  REQUIRE(rows < kIntLimit && rows * (I > I_s ? I : I_s) <= kIntLimit && T * k * H <= kIntLimit * 4L,
          "T*k*H or the SwiGLU buffer is too large");
  REQUIRE(H % dmoe::chunk_elems(dt) == 0, "H=%d must be a multiple of %d", H, dmoe::chunk_elems(dt));
  REQUIRE(H % 4 == 0, "H=%d must be a multiple of 4", H);
  if (routing == DMOE_ROUTE_TOPP) {
    REQUIRE(buf->coreset && buf->coreset_size, "Top-P routing needs coreset and coreset_size");
    REQUIRE(min_coreset >= k && min_coreset <= E, "min_coreset=%d must be in [k, E]", min_coreset);
    REQUIRE(top_p > 0.f && top_p <= 1.f, "p=%g must be in (0, 1]", static_cast<double>(top_p));
  }
  const size_t need = layer_workspace_bytes(n_blocks, block_size, H, E, I, I_s, k, dt);
  REQUIRE(buf->ws_bytes >= need, "workspace of %zu bytes is smaller than the %zu bytes needed", buf->ws_bytes, need);
  REQUIRE(!buf->res_out || buf->res_in, "res_out needs res_in");
  {
    // the residual's arrays are [T][H] of dt; res_out overlaps neither x nor y, res_in not y (it may be x)
    const size_t rb = static_cast<size_t>(T) * H * dmoe::dtype_bytes(dt);
    const size_t yb = static_cast<size_t>(T) * H * dmoe::dtype_bytes(y_dt);
    auto overlaps = [](const void* a, size_t na, const void* b, size_t nb) {
      const char* pa = static_cast<const char*>(a);
      const char* pb = static_cast<const char*>(b);
      return pa < pb + nb && pb < pa + na;
    };
    REQUIRE(!buf->res_out || (!overlaps(buf->res_out, rb, y, yb) && !overlaps(buf->res_out, rb, x, rb) &&
                              !overlaps(buf->res_in, rb, y, yb)),
            "res_out and res_in must not overlap x or y");
  }
  ALIGNED(x);
  ALIGNED(w_router);
  ALIGNED(bias);
  ALIGNED(w13);
  ALIGNED(w2);
  ALIGNED(ws13);
  ALIGNED(ws2);
  ALIGNED(y);
  ALIGNED(buf->logits);
  ALIGNED(buf->probs);
  ALIGNED(buf->x_chunked);
  ALIGNED(buf->block_scores);
  ALIGNED(buf->experts);
  ALIGNED(buf->combine_w);
  ALIGNED(buf->gap);
  ALIGNED(buf->coreset);
  ALIGNED(buf->coreset_size);
  ALIGNED(buf->slot_out);
  ALIGNED(buf->shared_out);
  ALIGNED(buf->workspace);
  ALIGNED(buf->res_in);
  ALIGNED(buf->res_out);
  ALIGNED(sched.n_unique);
  ALIGNED(sched.unique);
  ALIGNED(sched.offsets);
  ALIGNED(sched.scratch);
  ALIGNED(sched.row_token);
  ALIGNED(sched.row_slot);
  ALIGNED(sched.n_work);
  ALIGNED(sched.work);
  SUPPORT(E <= kMaxScheduleE, "the schedule supports E <= %d (E=%d)", kMaxScheduleE, E);
  if (dt == DMOE_BF16) {
    SUPPORT(H % 128 == 0 && I % 128 == 0 && I_s % 128 == 0,
            "bf16 layers need H, I and I_s to be multiples of 128 (H=%d, I=%d, I_s=%d)", H, I, I_s);
  }
  SUPPORT(buf->slot_fmt == DMOE_SLOT_F32 || dt == DMOE_BF16, "scaled-half slot outputs need a DMOE_BF16 layer");
  if (routing == DMOE_ROUTE_TOPP) {
    SUPPORT(dmoe::topp_supported(block_size, E, k), "the Top-P kernels do not support block_size=%d, E=%d, k=%d",
            block_size, E, k);
  }
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const int Ti = static_cast<int>(T);
  if (routing == DMOE_ROUTE_BLOCK && dmoe::layer_fused_fits(dt, n_blocks, Ti, H, E, I, I_s, k)) {
    dmoe::LayerArgs a{x, w_router, bias, w13, w2, ws13, ws2, Ti, H, E, I, I_s, k, buf->logits, buf->probs,
                      buf->x_chunked, buf->block_scores, buf->experts, buf->combine_w, buf->gap, sched,
                      buf->workspace, y, y_dt, buf->res_in, buf->res_out};
    return hip_status(dmoe::launch_layer_fused(a, s), __func__);
  }
  const size_t rbytes = dmoe::router_workspace_bytes(Ti, H, E, dt);
  void* ffn_ws = static_cast<char*>(buf->workspace) + align256(rbytes);
  dmoe::RouteArgs ra{x, w_router, bias, Ti, H, E, k, routing == DMOE_ROUTE_TOKEN ? 1 : block_size,
                     routing == DMOE_ROUTE_BLOCK, buf->logits, buf->probs, buf->x_chunked,
                     routing == DMOE_ROUTE_TOKEN ? nullptr : buf->block_scores, buf->experts, buf->combine_w,
                     buf->gap, sched, rbytes ? buf->workspace : nullptr, rbytes};
  if (routing == DMOE_ROUTE_TOPP) {
    ra.topp = true;
    ra.top_p = top_p;
    ra.min_coreset = min_coreset;
    ra.coreset = buf->coreset;
    ra.coreset_size = buf->coreset_size;
  }
  hipError_t err = dmoe::launch_route(ra, dt, s);
  if (err != hipSuccess) return hip_status(err, __func__);
  const long mw = routing == DMOE_ROUTE_BLOCK ? dmoe::schedule_max_work(n_blocks, block_size, k, E)
                                              : dmoe::schedule_max_work(T, 1, k, E);
  dmoe::FfnArgs fa{buf->x_chunked, x, w13, w2, ws13, ws2, Ti, H, E, I, I_s, k, static_cast<int>(mw), sched,
                   buf->slot_out, buf->slot_fmt, buf->shared_out, ffn_ws};
  err = dmoe::launch_ffn(fa, dt, s);
  if (err != hipSuccess) return hip_status(err, __func__);
  return hip_status(dmoe::launch_combine(buf->slot_out, buf->slot_fmt, buf->combine_w, buf->shared_out, y_dt, Ti, H,
                                         k, y, s, buf->res_in, buf->res_out, dt),
                    __func__);
}

}  // extern "C"
