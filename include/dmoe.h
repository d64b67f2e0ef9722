/*
 * dmoe.h -- C ABI of the block-routed MoE layer forward for AMD Instinct
 * MI355X (gfx950).
 *
 * One MoE layer forward of a block-diffusion decode step, split into the
 * steps of the routing procedure of "dMoE: dLLMs with Learnable Block
 * Experts" (Sec. 4.2 and Alg. 1) followed by expert execution:
 *
 *   dmoe_router_logits         token scores s_i = Router(t_i)  (Sec. 4.2)
 *   dmoe_block_aggregate_topk  block scores S_block = mean_i s_i, coreset
 *                              C = top-k(S_block), per-token weights
 *                              (Sec. 4.2 aggregation; Alg. 1 with |C| = k)
 *   dmoe_token_topk            token-level top-k (the "Original" routing of
 *                              Sec. 5.1, the baseline)
 *   dmoe_block_topp_route      Alg. 1 with its Top-P coreset: block scores from
 *                              each token's top-k, a shared coreset per block,
 *                              each token's top-k inside it
 *   dmoe_build_expert_schedule unique experts of the forward and the rows
 *                              (token, slot) that use each one (the unique
 *                              expert count of Sec. 3 is its n_unique)
 *   dmoe_expert_ffn            SwiGLU FFN of every unique expert over its
 *                              rows, plus the always-on shared expert
 *   dmoe_shared_expert_ffn     the shared expert alone (to overlap it with
 *                              the routing of the same forward)
 *   dmoe_combine               y_t = sum_j w[t,j] * FFN_{e_tj}(x_t) + FFN_s(x_t)
 *
 * dmoe_route_block / dmoe_route_token / dmoe_route_topp run the routing steps
 * and the schedule of one routing mode as one call with fewer kernel
 * launches; and two layout conversions for the expert FFN's operands:
 *
 *   dmoe_pack_expert_weights   expert weights -> the FFN's packed layout
 *                              (once, when the model is loaded)
 *   dmoe_pack_activations      hidden states -> chunk-major layout (also a
 *                              by-product of dmoe_router_logits)
 *
 * Chunk-major activations
 * -----------------------
 * The expert FFN reads hidden states as 16-byte chunks of c consecutive
 * features (c = 8 for DMOE_BF16, 4 for DMOE_F32), chunk-major:
 *   x_chunked[(j * T + t) * c + i] = x[t][j * c + i],   j < H/c, i < c
 * so that the same chunk of consecutive tokens is contiguous in memory.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every pointer argument is a DEVICE pointer (memory the caller allocated on
 *    the GPU, e.g. with hipMalloc or a torch CUDA tensor) unless the comment
 *    says otherwise.  The caller owns all memory.  The library allocates
 *    nothing and keeps no state between calls, except the per-GPU device
 *    array of dmoe_expert_ffn_noalloc.
 *  - All arrays are dense and row-major.  Matrices are indexed [row][col] with
 *    the last index contiguous.
 *  - Tokens are block-major: block b of a forward is rows
 *    [b*block_size, (b+1)*block_size) of the hidden states.
 *  - stream is a hipStream_t passed as void* (NULL = the null stream).  Every
 *    entry point only enqueues work on it and returns without synchronising;
 *    a fault inside a kernel surfaces at the caller's next synchronisation.
 *  - Ordering of a top-k: indices by (score descending, expert id ascending),
 *    so an exact tie goes to the lower expert id.
 *  - Errors: arguments are validated on the host before anything is launched.
 *      DMOE_ERR_INVALID_ARG  a required pointer is NULL, a size is out of range,
 *                            or a pointer is not aligned as documented;
 *      DMOE_ERR_UNSUPPORTED  valid arguments with no kernel (a shape outside
 *                            the documented limits);
 *      DMOE_ERR_HIP          a kernel launch failed.
 *    On a non-OK status nothing was enqueued (except for DMOE_ERR_HIP) and
 *    dmoe_last_error() describes the cause.
 *  - Element types: dmoe_dtype gives the storage type of hidden states,
 *    weights and the layer output.  Router logits, probabilities, block
 *    scores, combine weights and gaps are always float32; expert indices and
 *    schedules are int32.  Accumulation is float32 throughout.
 *  - Alignment: every pointer must be 16-byte aligned.
 */
#ifndef DMOE_H
#define DMOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum dmoe_status {
  DMOE_OK = 0,
  DMOE_ERR_INVALID_ARG = -1,
  DMOE_ERR_UNSUPPORTED = -2,
  DMOE_ERR_HIP = -3
} dmoe_status;

typedef enum dmoe_dtype {
  DMOE_F32 = 0,  /* IEEE binary32 */
  DMOE_BF16 = 1  /* bfloat16 (upper half of a binary32) */
} dmoe_dtype;

/*
 * Storage of the per-slot expert outputs slot_out [T][k][H] that
 * dmoe_expert_ffn writes and dmoe_combine reads (device memory, 16-byte
 * aligned, dmoe_slot_out_bytes(T, H, k, format) bytes):
 *   DMOE_SLOT_F32   float32 [T][k][H].
 *   DMOE_SLOT_F16S  scaled half, for DMOE_BF16 layers (about half the bytes
 *                   of the round trip through memory): uint16
 *                   half[T][k][H] (IEEE binary16 bit patterns), then int8
 *                   e[T][k][H/16]; value = half[t][j][h] * 2^e[t][j][h/16].
 *                   Each sixteen consecutive outputs share e, chosen so
 *                   that the largest finite magnitude of the sixteen lies in
 *                   [2^14, 2^15): no overflow, 11 significant bits
 *                   (relative error <= 2^-11) for every value within 2^28 of
 *                   that maximum, smaller ones with absolute error below
 *                   2^-25 of it; NaN and infinities are kept.  H % 16 == 0.
 */
typedef enum dmoe_slot_format {
  DMOE_SLOT_F32 = 0,
  DMOE_SLOT_F16S = 1
} dmoe_slot_format;

/* Bytes of slot_out for these sizes in format f (0 on invalid sizes). */
size_t dmoe_slot_out_bytes(int T, int H, int k, dmoe_slot_format f);

/*
 * Unique-expert schedule of one forward (device arrays, caller-allocated).
 * Written by dmoe_build_expert_schedule (or dmoe_route_*), read by
 * dmoe_expert_ffn.
 *   n_unique [1]        number of distinct experts selected in the forward
 *   unique   [E]        their ids, ascending, in unique[0 .. n_unique)
 *   offsets  [E + 1]    rows of unique[u] are rows offsets[u] .. offsets[u+1]
 *                       of row_token / row_slot; offsets[n_unique] = n_rows
 *   row_token[n_rows]   token of each row (n_rows = n_groups*group_size*k)
 *   row_slot [n_rows]   slot j in 0..k-1 of the token's expert list
 *   n_work   [1]        number of work items
 *   work     [4*max_work] work items {expert id, first row, row count, piece}:
 *                       each unique expert's rows cut, in order, into pieces
 *                       of at most DMOE_WORK_ROWS rows (piece = 0, 1, ... its
 *                       index within the expert); items are ordered by
 *                       expert id, then row.  max_work: dmoe_schedule_max_work.
 * Within one expert, rows are ordered by token.
 *   scratch  optional (NULL: not used); with group_size 1 and at least
 *            DMOE_SCHED_SPLIT_MIN entries (n_groups*k), a schedule with
 *            scratch is built by many workgroups instead of one; it needs
 *            (ceil(n_groups*k / 512) + 1) * E ints (dmoe_schedule_scratch_ints).
 *            The results are identical either way.
 */
#define DMOE_WORK_ROWS 128
#define DMOE_SCHED_SPLIT_MIN 2048

typedef struct dmoe_schedule {
  int32_t* n_unique;
  int32_t* unique;
  int32_t* offsets;
  int32_t* row_token;
  int32_t* row_slot;
  int32_t* n_work;
  int32_t* work;
  int32_t* scratch;
} dmoe_schedule;

/*
 * Upper bound of the schedule's work items for n_groups expert lists of k
 * experts over groups of group_size tokens (E experts): the capacity of
 * sched.work (in items of 4 int32) and the max_work argument of
 * dmoe_expert_ffn.  0 on invalid sizes.
 */
int dmoe_schedule_max_work(int n_groups, int group_size, int k, int E);

/* Ints of dmoe_schedule.scratch for n_groups expert lists of k among E
 * experts: (ceil(n_groups*k / 512) + 1) * E.  0 on invalid sizes. */
size_t dmoe_schedule_scratch_ints(int n_groups, int k, int E);

/*
 * Bytes of optional workspace that let dmoe_router_logits split the hidden
 * dimension over several workgroups (worth it when T is small: a decode
 * step).  0 when no split is used for these sizes.
 */
size_t dmoe_router_workspace_size(int T, int H, int E, dmoe_dtype dt);

/*
 * Router scores (Sec. 4.2, s_i = Router(t_i)): linear router and softmax.
 *   logits[t][e] = sum_h x[t][h] * w_router[e][h] + bias[e]
 *   probs[t][:]  = softmax(logits[t][:]) over all E experts (max-subtracted)
 * x [T][H] and w_router [E][H] of type dt; bias [E] float32 or NULL (no bias);
 * logits [T][E] float32 or NULL (not stored); probs [T][E] float32.
 * x_chunked: NULL, or T*H elements of type dt that receive x in the
 * chunk-major layout (see above; H must be a multiple of c), ready for
 * dmoe_expert_ffn; the router reads every chunk of x anyway.
 * workspace: NULL, or device scratch of ws_bytes >= dmoe_router_workspace_size
 * bytes (contents on entry do not matter; results do not depend on whether
 * it is given).  Calls sharing a workspace must not overlap in time.
 * Limits: T >= 1; 1 <= E <= 4096; H >= 1.  For DMOE_BF16: H % 128 == 0
 * (matrix-core tiles); DMOE_F32 has no further limit.
 */
dmoe_status dmoe_router_logits(const void* x, const void* w_router, const float* bias,
                               dmoe_dtype dt, int T, int H, int E, float* logits, float* probs,
                               void* x_chunked, void* workspace, size_t ws_bytes, void* stream);

/*
 * Block-level routing (Sec. 4.2 aggregation, Alg. 1 with a coreset of size k).
 * For each block b of block_size consecutive tokens:
 *   S[b][e]     = (1/block_size) * sum_{t in b} probs[t][e]   (token order)
 *   C_b         = top-k of S[b][:]                       -> block_experts[b][0..k)
 *   gap[b]      = S_(k) - S_(k+1)  (k-th minus (k+1)-th largest; +inf if k == E)
 *   w[t][j]     = probs[t][C_b[j]] / sum_j' probs[t][C_b[j']]   for t in b
 * probs [n_blocks*block_size][E]; block_scores [n_blocks][E] or NULL;
 * block_experts [n_blocks][k] int32; combine_w [n_blocks*block_size][k];
 * gap [n_blocks] or NULL.
 * Limits: n_blocks >= 1; 1 <= block_size <= 4096; 1 <= k <= min(E, 64);
 * E <= 4096.
 */
dmoe_status dmoe_block_aggregate_topk(const float* probs, int n_blocks, int block_size, int E,
                                      int k, float* block_scores, int32_t* block_experts,
                                      float* combine_w, float* gap, void* stream);

/*
 * Token-level top-k routing (the baseline): for each token t
 *   R_t = top-k of probs[t][:] -> token_experts[t][0..k)
 *   gap[t] = p_(k) - p_(k+1) (+inf if k == E)
 *   w[t][j] = probs[t][R_t[j]] / sum_j' probs[t][R_t[j']]
 * probs [T][E]; token_experts [T][k] int32; combine_w [T][k]; gap [T] or NULL.
 * Limits: T >= 1; 1 <= k <= min(E, 64); E <= 4096.
 */
dmoe_status dmoe_token_topk(const float* probs, int T, int E, int k, int32_t* token_experts,
                            float* combine_w, float* gap, void* stream);

/*
 * Alg. 1 of Sec. 4.2 with the Top-P coreset, on each block b of block_size
 * consecutive tokens:
 *   S[e]  = sum over the block's tokens, in token order, of TopKMask(probs[t], k)[e]
 *           (the token's own top-k probabilities, zeros elsewhere)
 *   Sn[e] = S[e] / sum_e' S[e']          (Normalize; the sum in expert-id order)
 *   C_b   = the shortest prefix of the experts ranked by Sn (desc, id asc) whose
 *           cumulative Sn, summed in that order in float32, reaches p; at least
 *           min_coreset experts                                  -> coreset[b]
 *   R_t   = top-k of probs[t] restricted to C_b                  -> token_experts[t]
 *   w[t][j] = probs[t][R_t[j]] / sum_j' probs[t][R_t[j']]
 * Every token of a block picks its own k experts inside the block's shared
 * coreset, so the unique experts of the block are at most |C_b|.
 * probs [n_blocks*block_size][E]; block_scores [n_blocks][E] (Sn) or NULL;
 * coreset [n_blocks][E] int32 (ids in rank order; the first coreset_size[b]
 * are C_b); coreset_size [n_blocks] int32; token_experts [T][k] int32;
 * combine_w [T][k]; gap [T] or NULL (k-th minus (k+1)-th probability inside
 * C_b; +inf if |C_b| == k).  Schedule token_experts with group_size = 1.
 * Limits: 1 <= k <= min(E, 64); k <= min_coreset <= E; 0 < p <= 1;
 * 1 <= block_size <= 4096.  Kernel limit (else DMOE_ERR_UNSUPPORTED): E <= 1024.
 */
dmoe_status dmoe_block_topp_route(const float* probs, int n_blocks, int block_size, int E, int k, float p,
                                  int min_coreset, float* block_scores, int32_t* coreset, int32_t* coreset_size,
                                  int32_t* token_experts, float* combine_w, float* gap, void* stream);

/*
 * Unique-expert schedule.  experts [n_groups][k] int32 holds one expert list
 * per group; group g covers tokens [g*group_size, (g+1)*group_size).  Block
 * routing passes block_experts with group_size = block_size; token routing
 * passes token_experts with group_size = 1.  The lists of a group must hold k
 * distinct ids in [0, E) (what the two top-k entry points produce); a
 * violation is not detected and yields an undefined schedule.
 * Writes every array of sched (see dmoe_schedule).
 * Limits: n_groups >= 1; group_size >= 1; 1 <= k <= min(E, 64); E <= 512;
 * n_groups*group_size*k < 2^31.
 */
dmoe_status dmoe_build_expert_schedule(const int32_t* experts, int n_groups, int group_size,
                                       int k, int E, dmoe_schedule sched, void* stream);

/*
 * The whole routing stage of one forward in one call, block-level:
 *   dmoe_router_logits(x, ..., logits, probs, x_chunked, workspace)
 *   dmoe_block_aggregate_topk(probs, n_blocks, block_size, E, k, ...)
 *   dmoe_build_expert_schedule(block_experts, n_blocks, block_size, k, E, sched)
 * with T = n_blocks*block_size, arguments as documented there, and results
 * bit-identical to that sequence.  A small forward (all T x E probabilities
 * fit in on-chip memory) runs as two kernels instead of four.
 * Limits: the union of the three calls' limits (E <= 512).
 */
dmoe_status dmoe_route_block(const void* x, const void* w_router, const float* bias, dmoe_dtype dt,
                             int n_blocks, int block_size, int H, int E, int k, float* logits,
                             float* probs, void* x_chunked, float* block_scores, int32_t* block_experts,
                             float* combine_w, float* gap, dmoe_schedule sched, void* workspace,
                             size_t ws_bytes, void* stream);

/*
 * The same for token-level routing (the baseline):
 *   dmoe_router_logits, dmoe_token_topk(probs, T, E, k, token_experts, ...),
 *   dmoe_build_expert_schedule(token_experts, T, 1, k, E, sched)
 * bit-identical to that sequence.
 */
dmoe_status dmoe_route_token(const void* x, const void* w_router, const float* bias, dmoe_dtype dt,
                             int T, int H, int E, int k, float* logits, float* probs, void* x_chunked,
                             int32_t* token_experts, float* combine_w, float* gap, dmoe_schedule sched,
                             void* workspace, size_t ws_bytes, void* stream);

/*
 * The same for Alg. 1 with the Top-P coreset (Sec. 4.2):
 *   dmoe_router_logits, dmoe_block_topp_route(probs, n_blocks, block_size, E,
 *   k, p, min_coreset, ...), dmoe_build_expert_schedule(token_experts,
 *   n_blocks*block_size, 1, k, E, sched)
 * bit-identical to that sequence (the router's softmax and every token's own
 * top-k run as one launch where the separate calls take two).
 * Limits: the union of the three calls' limits.
 */
dmoe_status dmoe_route_topp(const void* x, const void* w_router, const float* bias, dmoe_dtype dt, int n_blocks,
                            int block_size, int H, int E, int k, float p, int min_coreset, float* logits,
                            float* probs, void* x_chunked, float* block_scores, int32_t* coreset,
                            int32_t* coreset_size, int32_t* token_experts, float* combine_w, float* gap,
                            dmoe_schedule sched, void* workspace, size_t ws_bytes, void* stream);

/*
 * Hidden states x [T][H] (row-major, type dt) -> x_chunked [T*H] in the
 * chunk-major layout above.  For callers that do not run dmoe_router_logits
 * with its x_chunked output.  x and x_chunked must not overlap.
 * Limits: T, H >= 1; H % c == 0; T*H < 2^31.
 */
dmoe_status dmoe_pack_activations(const void* x, dmoe_dtype dt, int T, int H, void* x_chunked,
                                  void* stream);

/*
 * Expert weights in the layout dmoe_expert_ffn streams (call once when the
 * model is loaded; the FFN reads only the packed copies).
 * Inputs: w_gate, w_up [n_experts][I][H]; w_down [n_experts][H][I], type dt.
 * Outputs: w13 (2*n_experts*I*H elements) and w2 (n_experts*H*I elements) of
 * type dt; neither may overlap an input or the other.
 *   DMOE_BF16: matrix-core fragment order.  w13 holds, per expert, tiles of
 *     16 rows x 32 columns, index [it][ks] with it < I/8, ks < H/32; tile row
 *     r (r < 16) is the gate row (r%4 < 2) or the up row (r%4 >= 2) of
 *     intermediate unit 8*it + 2*(r/4) + r%2, columns 32*ks .. 32*ks+31.  w2
 *     holds, per expert, tiles [jt][ks] with jt < H/16, ks < I/32, tile row r
 *     being w_down row 16*jt + r, columns 32*ks .. 32*ks+31.  A tile is stored
 *     as 64 pieces of 8 elements; piece p = 16*g + r holds row r, columns
 *     8g .. 8g+7 of the tile.
 *   DMOE_F32: reduction-major.  w13[e][h][u] (u < 2*I) is w_gate[e][u][h]
 *     for u < I and w_up[e][u-I][h] otherwise; w2[e][i][j] = w_down[e][j][i].
 * The shared expert is packed by a second call with n_experts = 1, I = I_s.
 * Limits: n_experts, H, I >= 1; DMOE_BF16: H % 128 == 0 and I % 128 == 0.
 */
dmoe_status dmoe_pack_expert_weights(const void* w_gate, const void* w_up, const void* w_down,
                                     dmoe_dtype dt, int n_experts, int H, int I, void* w13, void* w2,
                                     void* stream);

/*
 * Bytes of workspace dmoe_expert_ffn needs for these sizes (the SwiGLU
 * activations of every routed row and every shared-expert row).
 * Returns 0 on invalid sizes.
 */
size_t dmoe_ffn_workspace_size(int T, int I, int I_s, int k, dmoe_dtype dt);

/*
 * Expert execution (Sec. 3: the MoE layer is routing plus expert execution;
 * each token's selected experts and the shared expert are SwiGLU FFNs): for
 * every unique expert e = sched.unique[u] and each of its rows (t, j):
 *   h = silu(W_gate[e] x_t) * (W_up[e] x_t)          (SwiGLU, silu(a) = a/(1+e^-a))
 *   slot_out[t][j][:] = W_down[e] h
 * and, when the shared expert is present (ws13 != NULL), for every token t:
 *   shared_out[t][:] = Ws_down (silu(Ws_gate x_t) * (Ws_up x_t))
 * Each selected expert's weights are streamed once per work item: an
 * expert's rows are cut into items of at most DMOE_WORK_ROWS, and an expert
 * with more rows than that (a popular expert, or the shared expert over more
 * than DMOE_WORK_ROWS tokens) is streamed once per item.
 * x_chunked: the hidden states x [T][H] in the chunk-major layout above.
 * x: the same hidden states row-major [T][H], optional (NULL: not used).
 * With it, bf16 rows whose tokens are not consecutive (token-level routing)
 * are read from x, one 64-byte piece per token and reduction step, instead
 * of four 16-byte chunks of x_chunked; results are identical either way.
 * w13, w2: all E routed experts packed by dmoe_pack_expert_weights (I);
 * ws13, ws2: the shared expert packed the same way (n_experts = 1, I = I_s),
 * both NULL with I_s == 0 or both set with I_s > 0.  All of type dt.
 * sched: written by dmoe_build_expert_schedule for these T and k.
 * max_work: at least dmoe_schedule_max_work(n_groups, group_size, k, E) of
 * the call that built sched.  The grid has max_work rows for the routed
 * experts; a work item past max_work is not run and its slot_out rows keep
 * what they held, so a smaller value gives wrong results without an error.
 * The shared expert's T rows are cut into pieces of DMOE_WORK_ROWS the same
 * way.
 * slot_out [T][k][H] in format slot_fmt (every (t, j) is written;
 * DMOE_SLOT_F16S only with DMOE_BF16, else DMOE_ERR_UNSUPPORTED); shared_out
 * [T][H] float32 (NULL iff no shared expert).
 * workspace: device scratch of at least dmoe_ffn_workspace_size(...) bytes,
 * ws_bytes its size.  Its contents on entry do not matter; calls that share
 * one workspace must not overlap in time (use one stream).
 * Limits: T >= 1; 1 <= k <= min(E, 64); E <= 512; 1 <= max_work <= T*k;
 * H % c == 0; (T*k + T) * max(I, I_s) < 2^31.
 * DMOE_BF16: H % 128 == 0, I % 128 == 0, I_s % 128 == 0 (matrix-core tiles).
 * DMOE_F32: any I, I_s >= 1.
 */
dmoe_status dmoe_expert_ffn(const void* x_chunked, const void* x, const void* w13, const void* w2,
                            const void* ws13, const void* ws2, dmoe_dtype dt, int T, int H, int E, int I,
                            int I_s, int k, int max_work, dmoe_schedule sched, void* slot_out,
                            dmoe_slot_format slot_fmt, float* shared_out, void* workspace, size_t ws_bytes,
                            void* stream);

/*
 * dmoe_expert_ffn without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture that may not call
 * hipMalloc, serving loops and harnesses that forbid allocation).  The
 * SwiGLU activations go to a device array of DMOE_NOALLOC_SCRATCH_BYTES that
 * the library holds on each GPU it runs on until the process ends; nothing
 * is allocated or freed by the call.  Arguments, results and limits are
 * those of dmoe_expert_ffn (results are bit-identical to it), plus:
 * dmoe_ffn_workspace_size(T, I, I_s, k, dt) must not exceed
 * DMOE_NOALLOC_SCRATCH_BYTES, else DMOE_ERR_INVALID_ARG and nothing is
 * enqueued.  Every call on one GPU shares that GPU's array and leaves its
 * contents behind (no part of it needs to start at zero): calls that overlap
 * in time on one GPU (two streams, two threads) race and must be serialised
 * by the caller.  DMOE_ERR_HIP if the array's device address cannot be found.
 */
#define DMOE_NOALLOC_SCRATCH_BYTES (16u << 20)
dmoe_status dmoe_expert_ffn_noalloc(const void* x_chunked, const void* x, const void* w13, const void* w2,
                                    const void* ws13, const void* ws2, dmoe_dtype dt, int T, int H, int E, int I,
                                    int I_s, int k, int max_work, dmoe_schedule sched, void* slot_out,
                                    dmoe_slot_format slot_fmt, float* shared_out, void* stream);

/*
 * The shared expert alone (the I_s > 0 part of dmoe_expert_ffn; expert
 * execution, Sec. 3, for the always-on shared expert): for every token t,
 *   shared_out[t][:] = Ws_down (silu(Ws_gate x_t) * (Ws_up x_t))
 * It needs no routing, so a caller can run it on a second stream while the
 * routing of the same forward runs, then call dmoe_expert_ffn with the
 * shared expert left out (ws13 = ws2 = shared_out = NULL, I_s = 0); the
 * results are those of one dmoe_expert_ffn call with the shared expert, up
 * to the fp32 summation order (the two calls may tile its rows differently).
 * x_chunked [T][H] chunk-major (see above); ws13, ws2: the shared expert
 * packed by dmoe_pack_expert_weights (n_experts = 1, I = I_s); shared_out
 * [T][H] float32.  workspace: device scratch of at least
 * dmoe_shared_ffn_workspace_size(T, I_s, dt) bytes (contents on entry do
 * not matter), not shared with a concurrent call.
 * Limits: T, H, I_s >= 1; H % c == 0; DMOE_BF16: H % 128 == 0 and
 * I_s % 128 == 0.
 */
size_t dmoe_shared_ffn_workspace_size(int T, int I_s, dmoe_dtype dt);
dmoe_status dmoe_shared_expert_ffn(const void* x_chunked, const void* ws13, const void* ws2, dmoe_dtype dt, int T,
                                   int H, int I_s, float* shared_out, void* workspace, size_t ws_bytes,
                                   void* stream);

/*
 * Weighted combine (Sec. 3, the layer output as the weighted sum of the
 * selected experts' outputs plus the shared expert's):
 *   y[t][h] = sum_{j=0..k-1} combine_w[t][j] * slot_out[t][j][h]  (+ shared_out[t][h])
 * summed in slot order in float32, stored as dt.  The weights are those the
 * routing entry points write: the token's own router probabilities on its
 * selected experts renormalised to sum to 1, with no further scaling (the
 * paper leaves the weighting open; this is the reading taken), and the
 * shared expert enters with weight 1.
 * slot_out [T][k][H] in format slot_fmt (scaled half values are decoded
 * exactly to float32 first); combine_w [T][k] float32; shared_out [T][H]
 * float32 or NULL; y [T][H] of type dt.
 * Limits: T >= 1; 1 <= k <= 64; H >= 1; H % 4 == 0 (DMOE_SLOT_F16S: H % 16 == 0).
 */
dmoe_status dmoe_combine(const void* slot_out, dmoe_slot_format slot_fmt, const float* combine_w,
                         const float* shared_out, dmoe_dtype dt, int T, int H, int k, void* y, void* stream);

/*
 * The whole MoE layer forward in one call: routing (dmoe_routing), the
 * expert FFN and the combine,
 *   y[t] = sum_j w[t][j] * FFN_{e_tj}(x_t) + FFN_shared(x_t)          (Sec. 3)
 * with the routing of Sec. 4.2 (block: Alg. 1 with a coreset of size k;
 * token: the baseline; topp: Alg. 1 with the Top-P coreset p, min_coreset).
 *
 * A block-routed forward of a single bf16 block (n_blocks == 1, block_size
 * <= 64, E <= 512 and E % 4 == 0, k + (I_s > 0) <= 12, H % 256 == 0, T*E
 * small enough for on-chip probabilities; dmoe_moe_forward_fused says
 * whether a call qualifies) runs as three kernels: the router (partial
 * logits over up to four slices of the hidden dimension, and x in the
 * chunk-major layout); the routing, recomputed by every workgroup of
 * the routed gate/up (the combine weight applied to the SwiGLU
 * activations), with the shared expert's gate/up as further workgroups of
 * the same launch; and one down projection over all selected experts and
 * the shared expert that writes y (no slot outputs, no combine kernel).  Its routing outputs equal
 * dmoe_route_block's up to the float32 rounding of the logits (the two
 * routers may split the hidden dimension differently), and y
 * differs from the chained path's by the bf16 rounding of the weighted
 * activations.  Every other forward chains dmoe_route_block / _token /
 * _topp, dmoe_expert_ffn and dmoe_combine, with results bit-identical to
 * those calls.
 *
 * Inputs: x [T][H] (T = n_blocks*block_size); w_router [E][H]; bias [E] or
 * NULL; w13, w2 routed and ws13, ws2 shared experts packed by
 * dmoe_pack_expert_weights (ws13 = ws2 = NULL iff I_s == 0); all of type dt.
 * buf: a HOST pointer to the device buffers below, all as documented for the
 * entry points the layer chains (experts is block_experts [n_blocks][k] for
 * block routing and token_experts [T][k] otherwise; gap is [n_blocks] or
 * [T]; coreset and coreset_size are used by topp only, else may be NULL;
 * slot_out [T][k][H] (format slot_fmt) and shared_out [T][H] are scratch
 * of the chained path and are left untouched by the three-kernel path,
 * shared_out NULL iff I_s == 0).  y [T][H] of type y_dt.  workspace: at least
 * dmoe_moe_forward_workspace_size bytes (contents on entry do not matter;
 * calls sharing one must not overlap in time).
 * Residual (optional, for chaining layers: the next layer's input is a base
 * stream plus this layer's output): with res_out set, the forward also
 * writes res_out[t][h] = round_dt(res_in[t][h] + y[t][h]), y taken in
 * float32 before its own rounding to y_dt, both [T][H] of type dt; res_in
 * must then be set too.  res_out may overlap neither x nor y (it is written
 * while they are read); res_in may be x itself but must not overlap y.  The three-kernel
 * path writes it from the down projection's epilogue and the chained path
 * from the combine, so no further kernel runs.  res_out NULL: not written.
 * Limits: those of the chained entry points (E <= 512; bf16: H, I, I_s
 * multiples of 128).
 */
typedef enum dmoe_routing {
  DMOE_ROUTE_BLOCK = 0,
  DMOE_ROUTE_TOKEN = 1,
  DMOE_ROUTE_TOPP = 2
} dmoe_routing;

typedef struct dmoe_layer_buffers {
  float* logits;        /* [T][E] or NULL */
  float* probs;         /* [T][E] */
  void* x_chunked;      /* T*H elements of dt */
  float* block_scores;  /* [n_blocks][E] or NULL */
  int32_t* experts;
  float* combine_w;     /* [T][k] */
  float* gap;           /* or NULL */
  int32_t* coreset;     /* topp: [n_blocks][E] */
  int32_t* coreset_size;/* topp: [n_blocks] */
  dmoe_schedule sched;
  void* slot_out;       /* [T][k][H] in format slot_fmt */
  dmoe_slot_format slot_fmt;
  float* shared_out;
  void* workspace;
  size_t ws_bytes;
  const void* res_in;   /* [T][H] of dt, or NULL (no residual output) */
  void* res_out;        /* [T][H] of dt: round_dt(res_in + y), or NULL */
} dmoe_layer_buffers;

/* Bytes of dmoe_layer_buffers.workspace for these sizes (0 on invalid sizes). */
size_t dmoe_moe_forward_workspace_size(int n_blocks, int block_size, int H, int E, int I, int I_s, int k,
                                       dmoe_dtype dt);

/*
 * 1 if dmoe_moe_forward with these arguments runs the three-kernel path of a
 * single block (see above), 0 if it chains the entry points (also for sizes
 * dmoe_moe_forward would reject).  Host only; enqueues nothing.
 */
int dmoe_moe_forward_fused(dmoe_dtype dt, int n_blocks, int block_size, int H, int E, int I, int I_s, int k,
                           dmoe_routing routing);

dmoe_status dmoe_moe_forward(const void* x, const void* w_router, const float* bias, const void* w13,
                             const void* w2, const void* ws13, const void* ws2, dmoe_dtype dt, int n_blocks,
                             int block_size, int H, int E, int I, int I_s, int k, dmoe_routing routing, float top_p,
                             int min_coreset, const dmoe_layer_buffers* buf, void* y, dmoe_dtype y_dt,
                             void* stream);

/* Message describing the last non-OK status returned on this thread ("" if none). */
const char* dmoe_last_error(void);

/* Library version, e.g. "0.1.0" (host string, owned by the library). */
const char* dmoe_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DMOE_H */
