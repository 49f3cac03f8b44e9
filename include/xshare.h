/*
 * xshare.h -- C ABI of the XShare batch-level MoE layer for AMD Instinct MI355X (gfx950).
 *
 * XShare (arXiv 2602.07265) picks ONE shared expert set S for a whole decode batch by
 * maximising the total gating score of the selected experts under a budget (Section 3.2,
 * Eq. (2); greedy is optimal by Proposition 3.1 / Corollary 3.2), then routes every token to
 * its top-k experts inside S (Algorithm 2), so that only the weights of experts in S are
 * read.  For speculative-decoding batches the set is built per request first and then
 * completed at batch level (Section 4.1, Algorithms 3 and 4).  Under expert parallelism the
 * experts are spread over G GPU groups and the set is grown one expert per group in turn,
 * which bounds the most loaded group (Section 5, Eq. (5), Algorithms 5 and 6).  The whole
 * layer of Section 2.1 is available too: router logits h = W_g x on the device, the routed
 * experts of the selected set, and always-on shared experts.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - All array arguments are DEVICE pointers owned by the caller; the parameter structs are
 *   HOST pointers read during the call only.  The library never allocates, frees or keeps a
 *   pointer after returning; scratch memory comes from the caller's workspace `ws`
 *   (size from the matching *_workspace_bytes function, 256-byte aligned).
 * - Calls are asynchronous and stream-ordered on `stream` (a hipStream_t; NULL = the
 *   default stream).  Outputs are valid once the stream has reached the end of the call.
 *   Nothing is copied back to the host and the stream is never synchronised.  A call only
 *   launches kernels (no memset, copy or allocation), so it can be captured in a HIP graph
 *   and replayed with the same pointers; calls that share a workspace must be ordered.
 * - Host-checkable errors are returned before anything is enqueued: XSHARE_EINVAL for an
 *   invalid argument, XSHARE_EUNSUPPORTED for a valid size outside the kernels' limits,
 *   XSHARE_EWORKSPACE when ws_bytes is too small.  XSHARE_EHIP reports a failed launch.
 * - Logits must be finite; NaN or infinity is not detected on the device and gives
 *   unspecified (but memory-safe) results.
 * - Selection is deterministic and bit-identical to the fp32 recipe documented below:
 *   logits are canonicalised with h + 0.0 (so -0.0 == +0.0); every ranking uses the key
 *   (value descending, expert index ascending); gates are the softmax over a token's k
 *   chosen logits (Section 2.2) computed as e_r = exp(h_r - h_0) with a fixed fp32
 *   exponential (Cody-Waite reduction by ln 2, degree-7 Taylor polynomial, no fused
 *   multiply-add, 0 below -80), Z summed left to right in rank order, g_r = e_r / Z
 *   correctly rounded; batch scores s_j = sum_i g_ij are summed in ascending token order.
 *
 * Limits: 1 <= N <= 1024, 1 <= k <= min(N, 32), 0 <= T <= 4096, T*k <= 8192;
 * d and f multiples of 32 (xshare_moe_forward).
 */
#ifndef XSHARE_H
#define XSHARE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  XSHARE_OK = 0,
  XSHARE_EINVAL = 1,        /* invalid argument: range, null pointer, alignment, offsets   */
  XSHARE_EUNSUPPORTED = 2,  /* valid, but outside the limits listed above                  */
  XSHARE_EWORKSPACE = 3,    /* ws is NULL or ws_bytes < the required workspace size         */
  XSHARE_EHIP = 4           /* a HIP launch failed (hipGetLastError after enqueue)          */
} xshare_status;

/* How `budget` is read (the paper uses both readings of m_l).                             */
enum {
  XSHARE_BUDGET_TOTAL = 0,  /* |S| <= budget; requires budget >= k                          */
  XSHARE_BUDGET_EXTRA = 1,  /* budget experts are added beyond the warm-up set (flat) or     *
                             * beyond the union of the per-request sets (hierarchical), as   *
                             * in the paper's (m_l, k0) settings of Section 6                */
  XSHARE_BUDGET_PER_GROUP = 2, /* budget is m_g, experts per GPU group (Algorithm 5); only   *
                             * with an xshare_ep_layout, which in turn requires this mode    */
  XSHARE_BUDGET_THRESHOLD = 3 /* Algorithm 1's own rule: add experts while                   *
                             * f(S) < threshold * f(E), f = summed batch score (Eq. (2));    *
                             * |S| adapts to the batch; `budget` is ignored (>= 0)           */
};

/* Which gates g_ij enter the scores s_j = sum_i g_ij (Eq. (2)).                            */
enum {
  XSHARE_SCORE_TOPK = 0,    /* top-k-sparse renormalised gates of Section 2.2 (default);    *
                             * candidates are the experts some token has in its top-k        */
  XSHARE_SCORE_DENSE = 1    /* softmax over all N experts (max-shifted, summed in index     *
                             * order); every expert is a candidate                           */
};

/*
 * Running totals over the MoE layers of one forward pass (Section 3.2: the layers share a
 * global budget K, sum_l |S_l| <= K).  DEVICE memory owned by the caller, who zeroes it at
 * the start of a pass; each call whose params name it adds its own counts at the end of its
 * selection kernel (one thread, a plain read-modify-write: calls that share a ledger must
 * be ordered, e.g. issued on one stream).
 */
typedef struct {
  int32_t layers;           /* calls that added to the ledger                               */
  int32_t selected;         /* sum of |S_l|                                                 */
  int32_t active;           /* sum of the experts whose weights the calls streamed          */
  int32_t vanilla_union;    /* sum of |U_l|: what plain top-k routing would have activated  */
  int32_t invalid;          /* calls that selected nothing (invalid offsets or group map)   */
  int32_t max_selected;     /* largest |S_l| of a call                                      */
  int32_t reserved[2];
} xshare_budget_ledger;

typedef struct {
  int32_t n_experts;          /* N: routed experts of the layer                             */
  int32_t top_k;              /* k: experts per token (Section 2.2)                         */
  int32_t warmup_k0;          /* k0: top-k0 of every token always enters S (0 <= k0 <= k)   */
  int32_t budget;             /* M: see XSHARE_BUDGET_*                                    */
  int32_t budget_mode;        /* XSHARE_BUDGET_TOTAL, _EXTRA or _PER_GROUP                  */
  int32_t score_mode;         /* XSHARE_SCORE_TOPK or XSHARE_SCORE_DENSE                    */
  int32_t per_request_budget; /* m_r (Algorithm 3); read by the hierarchical calls only     */
  float threshold;            /* tau >= 0, finite; read in XSHARE_BUDGET_THRESHOLD mode only: *
                               * f(E) = sum of every s_j in index order, f(S) = the starting  *
                               * set's scores in ranking order, then each added expert's, all *
                               * fp32; the target tau * f(E) is one fp32 product; the starting *
                               * set is never cut; tau > 1 takes every candidate              */
  xshare_budget_ledger* ledger; /* nullable DEVICE: this call's counts are added to it       */
} xshare_route_params;

/* Per-call statistics, written to DEVICE memory by the kernels.                          */
typedef struct {
  int32_t n_selected;       /* |S|                                                        */
  int32_t n_active;         /* experts with at least one routed token (weights streamed);  *
                             * with a local group, only that group's experts                */
  int32_t n_vanilla_union;  /* |U|, U = union of every token's plain top-k (Section 3.1)    */
  int32_t n_warmup;         /* |S_0|, S_0 = union of every token's top-k0                   */
  int32_t n_start;          /* size of the set the batch greedy starts from: |S_0| (flat),  *
                             * |union_r S_r| (hierarchical)                                 */
  int32_t budget_eff;       /* effective set size the greedy fills to (clamped to [k, |C|]); *
                             * min(m_g * G, N) for the expert-parallel selection            */
  int32_t max_group_load;   /* MaxLoad(S) = max_g |S on group g| (Section 5.1); 0 without   *
                             * GPU groups                                                    */
  int32_t reserved;
} xshare_stats;

/*
 * Placement of the experts over G GPU groups for expert parallelism (Section 5.1): the
 * groups partition the experts, E = E_1 u ... u E_G.
 *
 *   n_groups          G, 1 <= G <= N.
 *   expert_group      DEVICE [N] int32, group of expert j in [0, G); NULL = equal contiguous
 *                     blocks, expert j in group j / (N / G) (then G must divide N).  Entries
 *                     outside [0, G) are detected on the device: the call then selects
 *                     nothing, writes ids -1 and weights 0, and stats->n_selected = -1.
 *   host_expert_group nullable HOST copy of expert_group, validated before launch when given.
 *   local_group       xshare_moe_forward only: -1 computes the whole layer; g in [0, G)
 *                     computes one GPU group's share, y_i = sum of w_ir * E_{e_ir}(x_i) over
 *                     the ranks r whose expert is on group g, reading only that group's
 *                     weights (the shares of all groups sum to the layer output).
 */
typedef struct {
  int32_t n_groups;
  int32_t local_group;
  const int32_t* expert_group;
  const int32_t* host_expert_group;
} xshare_ep_layout;

/*
 * Always-on shared experts (Section 2.1: y gains sum_s E^s_s(x) with weight 1).  Each has
 * the routed experts' shape, SwiGLU with hidden width f; a wider shared expert of width
 * m * f is m of these holding slices of its hidden units (the hidden units of a SwiGLU are
 * independent, so the sum is the same function).
 *
 *   n_shared  N_s, 0 <= N_s <= 64 (more: XSHARE_EUNSUPPORTED).
 *   w1, w3    DEVICE [N_s, f, d] bf16; w2 DEVICE [N_s, d, f] bf16; 16-byte aligned.
 */
typedef struct {
  int32_t n_shared;
  const uint16_t* w1;
  const uint16_t* w3;
  const uint16_t* w2;
} xshare_shared_experts;

/* Workspace for xshare_route / xshare_select_hier with T tokens (bytes, 256-aligned).    */
size_t xshare_route_workspace_bytes(int32_t T, const xshare_route_params* params);

/* Workspace for xshare_moe_forward (includes the routing workspace); `ep` and `shared` as *
 * passed to xshare_moe_forward (nullable).  Returns 0 for invalid arguments.              */
size_t xshare_moe_workspace_bytes(int32_t T, int32_t d, int32_t f,
                                  const xshare_route_params* params, const xshare_ep_layout* ep,
                                  const xshare_shared_experts* shared);

/* Workspace for xshare_moe_layer: that of xshare_moe_forward plus the router's scratch    *
 * and a [T, N] fp32 logits buffer.                                                        */
size_t xshare_layer_workspace_bytes(int32_t T, int32_t d, int32_t f,
                                    const xshare_route_params* params,
                                    const xshare_ep_layout* ep,
                                    const xshare_shared_experts* shared);

/* Workspace for xshare_router_logits (bytes, 256-aligned: fp32 partial sums over parts of *
 * d); 0 for invalid sizes.                                                                */
size_t xshare_router_workspace_bytes(int32_t T, int32_t d, int32_t n_experts);

/*
 * xshare_router_logits -- router logits h = W_g x of a batch (Section 2.2).
 *
 *   x        [T, d] bf16 row-major, 16-byte aligned.
 *   w_gate   [N, d] bf16 (nn.Linear [out, in]), 16-byte aligned; N = n_experts <= 1024.
 *   logits   out [T, N] fp32: h_ij = sum_q x_iq * W_g[j, q]; the bf16 products are exact in
 *            fp32 and accumulated in fp32 (matrix-core blocks of 32 within parts of d; the
 *            parts' sums added in part order), so
 *            |h - exact| <= d * 2^-24 * sum_q |x_iq W_g[j, q]| (up to second order) and
 *            repeated calls give identical bits.
 *   d        multiple of 32.
 */
xshare_status xshare_router_logits(const uint16_t* x, const uint16_t* w_gate, int32_t T,
                                   int32_t d, int32_t n_experts, float* logits, void* ws,
                                   size_t ws_bytes, hipStream_t stream);

/*
 * xshare_route -- batch-aware expert selection for one layer (Algorithm 2, Section 3.4).
 *
 *   logits    [T, N] fp32 row-major: router logits h = W_g x of the batch (Section 2.2).
 *   T         number of tokens in the batch (0 allowed: S is empty).
 *   sel_mask  out [N] uint8: 1 if expert j is in S, else 0.
 *   topk_ids  out [T, k] int32: token i's top-k experts inside S, rank order (refinement).
 *   topk_w    out [T, k] fp32: their gates, softmax renormalised over those k.
 *   stats     out, nullable: one xshare_stats.
 *
 * Steps: warm-up S_0 = union of top-k0; budgeted greedy on s_j (Algorithm 1 with the
 * fixed budget of Section 3.4; a warm-up set larger than a total budget is cut by score);
 * refinement.
 */
xshare_status xshare_route(const float* logits, int32_t T, const xshare_route_params* params,
                           uint8_t* sel_mask, int32_t* topk_ids, float* topk_w,
                           xshare_stats* stats, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * xshare_select_hier -- speculative-decoding-aware selection (Algorithms 3 and 4, Section 4.1).
 *
 *   req_offsets  [R + 1] int32, DEVICE: request r owns tokens [o_r, o_{r+1});
 *                must satisfy 0 = o_0 < o_1 < ... < o_R = T.  Violations are detected on
 *                the device: the call then selects nothing, writes ids -1 and weights 0,
 *                and stats->n_selected = -1.  Pass host_offsets to have them rejected
 *                before launch instead.
 *   host_offsets nullable HOST copy of req_offsets, validated when given.
 *   R            number of requests (0 only with T == 0).
 *   Other arguments as xshare_route; params->per_request_budget is m_r.
 *
 * Per request r: S_r = S_0(r) plus the m_r best remaining experts of r by the request's own
 * score (Eq. (3)); then S = GreedySelect over the batch score (Eq. (4)) starting from the
 * union of the S_r (warm-up experts first when a total budget cuts it); refinement.
 */
xshare_status xshare_select_hier(const float* logits, int32_t T, const int32_t* req_offsets,
                                 const int32_t* host_offsets, int32_t R,
                                 const xshare_route_params* params, uint8_t* sel_mask,
                                 int32_t* topk_ids, float* topk_w, xshare_stats* stats,
                                 void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * xshare_select_ep -- expert-parallelism-aware selection (Algorithms 5 and 6, Section 5).
 *
 *   ep          HOST pointer to the group layout (local_group is ignored here).
 *   params      budget_mode must be XSHARE_BUDGET_PER_GROUP; budget is m_g >= 0.
 *   group_load  out, nullable: DEVICE [G] int32, Load_g(S) = |S on group g|.
 *   Other arguments as xshare_route (workspace from xshare_route_workspace_bytes).
 *
 * Starting from the warm-up set S_0, rounds in which every group in turn adds its best
 * remaining candidate (score descending, index ascending), while |S| < m_g * G at the start
 * of a round.  A group whose load (warm-up experts included) has reached m_g adds nothing
 * more (the constraint of Eq. (5)); a group without candidates is skipped; a round that
 * adds nothing ends the loop.  The warm-up set is never cut, so a group can exceed m_g
 * through S_0 alone.  If fewer than k experts result, the best remaining candidates are
 * added regardless of group, so that every token keeps k experts.  Then refinement.
 */
xshare_status xshare_select_ep(const float* logits, int32_t T, const xshare_route_params* params,
                               const xshare_ep_layout* ep, uint8_t* sel_mask, int32_t* topk_ids,
                               float* topk_w, int32_t* group_load, xshare_stats* stats,
                               void* ws, size_t ws_bytes, hipStream_t stream);

/* Stage boundaries recorded by xshare_moe_forward when stage_events is given.            */
#define XSHARE_N_STAGE_EVENTS 5  /* start | route | gate-up GEMM | down GEMM | combine end */

/*
 * xshare_moe_forward -- the whole routed-expert MoE layer for one decode batch.
 *
 *   x        [T, d] bf16 (uint16 bit patterns) row-major: token hidden states.
 *   logits   [T, N] fp32: router logits.
 *   w1, w3   [N, f, d] bf16: gate and up projections of every expert, nn.Linear [out, in].
 *   w2       [N, d, f] bf16: down projections.
 *   req_offsets/host_offsets/R: as xshare_select_hier, or req_offsets == NULL for the flat
 *            selection of xshare_route.
 *   ep       nullable HOST pointer: the expert-parallel selection of xshare_select_ep and,
 *            with ep->local_group >= 0, one group's share of y (see xshare_ep_layout).
 *            Not combined with req_offsets (XSHARE_EUNSUPPORTED).
 *   shared   nullable HOST pointer: always-on shared experts, added to y after the routed
 *            terms with weight 1 (not with a local group: XSHARE_EUNSUPPORTED).
 *   y        out [T, d] bf16: y_i = sum_r w_ir * E_{e_ir}(x_i) with the refined routing
 *            (Section 2.1 without the shared-expert term), E(x) = W2 (silu(W1 x) * (W3 x)),
 *            fp32 accumulation, rounded to bf16 (nearest even) once at the end.
 *   sel_mask, topk_ids, topk_w, stats: nullable copies of the routing outputs.
 *   stage_events: nullable; XSHARE_N_STAGE_EVENTS hipEvent_t handles created by the caller,
 *            recorded on `stream` at the stage boundaries (profiling).
 *
 * Only the weights of experts that receive at least one token are read, each once per
 * (up to) 32 tokens routed to it.  Pointers x, w1, w3, w2 and y must be 16-byte aligned.
 * With shared experts, y_i = sum_r w_ir * E_{e_ir}(x_i) + sum_s E^s_s(x_i), the shared
 * terms added after the routed ones.
 */
xshare_status xshare_moe_forward(const uint16_t* x, const float* logits, int32_t T, int32_t d,
                                 int32_t f, const uint16_t* w1, const uint16_t* w3,
                                 const uint16_t* w2, const xshare_route_params* params,
                                 const int32_t* req_offsets, const int32_t* host_offsets,
                                 int32_t R, const xshare_ep_layout* ep,
                                 const xshare_shared_experts* shared, uint16_t* y,
                                 uint8_t* sel_mask, int32_t* topk_ids, float* topk_w,
                                 xshare_stats* stats, void* ws, size_t ws_bytes,
                                 void* const* stage_events, hipStream_t stream);

/* Weight formats of the routed experts (xshare_layer_args.weight_format).                  */
enum {
  XSHARE_WEIGHTS_BF16 = 0,  /* w1, w3 [N, f, d] and w2 [N, d, f] bf16; no scales             */
  XSHARE_WEIGHTS_FP8 = 1,   /* as xshare_moe_forward_fp8: E4M3FN codes, fp32 row scales      */
  XSHARE_WEIGHTS_MXFP4 = 2  /* as xshare_moe_forward_mxfp4: E2M1 codes, tiled E8M0 scales     */
};

/*
 * Every argument of a layer call, for xshare_moe_forward_v2.  The fixed-signature layer
 * calls (xshare_moe_forward, _fp8, _mxfp4, xshare_moe_layer) fill one of these and run the
 * same code.  Zero-initialise it, set struct_size = sizeof(xshare_layer_args), then the
 * fields the call uses; pointer conventions as in those calls.
 *
 *   x, T, d, f        hidden states [T, d] bf16 and the layer's sizes.
 *   logits / w_gate   exactly one when T > 0: fp32 router logits [T, N] (xshare_moe_forward),
 *                     or bf16 router weights [N, d], the logits then computed on the device
 *                     (xshare_moe_layer; logits_out optionally receives them).
 *   weight_format     XSHARE_WEIGHTS_*; w1, w3, w2 and the three scale arrays as the
 *                     matching fixed-signature call takes them (scales NULL for bf16).
 *   params, req_offsets / host_offsets / R, ep, shared: as xshare_moe_forward (shared
 *                     experts with bf16 weights only).
 *   y, sel_mask, topk_ids, topk_w, stats: outputs as xshare_moe_forward.
 *   ws, ws_bytes      workspace of xshare_moe_forward_v2_workspace_bytes bytes.
 *   stage_events, stream: as xshare_moe_forward.
 */
typedef struct {
  size_t struct_size;
  int32_t T, d, f;
  const uint16_t* x;
  const float* logits;
  const uint16_t* w_gate;
  int32_t weight_format;
  const void* w1;
  const void* w3;
  const void* w2;
  const void* w1_scale;
  const void* w3_scale;
  const void* w2_scale;
  const xshare_route_params* params;
  const int32_t* req_offsets;
  const int32_t* host_offsets;
  int32_t R;
  const xshare_ep_layout* ep;
  const xshare_shared_experts* shared;
  uint16_t* y;
  float* logits_out;
  uint8_t* sel_mask;
  int32_t* topk_ids;
  float* topk_w;
  xshare_stats* stats;
  void* ws;
  size_t ws_bytes;
  void* const* stage_events;
  hipStream_t stream;
} xshare_layer_args;

/* Workspace of xshare_moe_forward_v2 for these arguments (sizes, modes, ep, shared, whether *
 * w_gate is given); 0 if they are invalid.                                                   */
size_t xshare_moe_forward_v2_workspace_bytes(const xshare_layer_args* args);

/*
 * xshare_moe_forward_v2 -- the MoE layer of Sections 2.1-5 (selection by Algorithm 2, 3-4 or
 * 5-6, the selected routed experts, the shared experts, combine) from one argument struct.
 * XSHARE_EINVAL also for a struct_size other than sizeof(xshare_layer_args), both or neither
 * of logits and w_gate (T > 0), or an unknown weight format.
 */
xshare_status xshare_moe_forward_v2(const xshare_layer_args* args);

/* Size of the scratch array that xshare_moe_forward_noalloc uses on each GPU (64 MiB).     */
#define XSHARE_NOALLOC_SCRATCH_BYTES (64u << 20)

/*
 * xshare_moe_forward_noalloc -- xshare_moe_forward for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same layer, the same kernels and the same results, with no workspace
 * argument.  Its scratch is a fixed array of XSHARE_NOALLOC_SCRATCH_BYTES inside the
 * library, one per GPU, which that GPU holds from the first call on it until the process
 * ends.  Nothing is allocated or freed, by the library or any library it calls.
 *
 *   Arguments as xshare_moe_forward, without ws / ws_bytes.
 *   Limit: xshare_moe_workspace_bytes(T, d, f, params, ep, shared) <= the array's size
 *          (for instance the DeepSeek-R1 shape, d = 7168, f = 2048, N = 256, k = 8, up to
 *          T = 64 under a total budget); larger calls return XSHARE_EWORKSPACE before
 *          anything is enqueued.
 *   The array used is the current device's; a non-NULL stream must belong to it
 *   (XSHARE_EINVAL otherwise).  XSHARE_EHIP if its address cannot be obtained.
 *   Every call on one GPU shares that GPU's array and it keeps the last call's contents (no
 *   kernel reads scratch it has not written in the same call, so nothing needs clearing).
 *   Calls that overlap on one GPU -- on different streams, or from threads without an
 *   ordering between them -- race on the array and give wrong results: order them, e.g. on
 *   one stream.
 */
xshare_status xshare_moe_forward_noalloc(const uint16_t* x, const float* logits, int32_t T,
                                         int32_t d, int32_t f, const uint16_t* w1,
                                         const uint16_t* w3, const uint16_t* w2,
                                         const xshare_route_params* params,
                                         const int32_t* req_offsets,
                                         const int32_t* host_offsets, int32_t R,
                                         const xshare_ep_layout* ep,
                                         const xshare_shared_experts* shared, uint16_t* y,
                                         uint8_t* sel_mask, int32_t* topk_ids, float* topk_w,
                                         xshare_stats* stats, void* const* stage_events,
                                         hipStream_t stream);

/*
 * xshare_moe_forward_fp8 -- xshare_moe_forward with FP8 routed-expert weights (half the
 * bytes of bf16 on the stream that bounds the layer; the paper is silent on precision).
 *
 *   w1, w3    [N, f, d] uint8: OCP FP8 E4M3FN codes (1 sign, 4 exponent bits with bias 7,
 *             3 mantissa bits; 0x7F and 0xFF are NaN and must not occur), 16-byte aligned.
 *   w2        [N, d, f] uint8, same format.
 *   w1_scale, w3_scale  [N, f] fp32; w2_scale [N, d] fp32: one scale per output row, the
 *             weight being decode(code) * scale.  Codes are decoded exactly to bf16 and the
 *             row scale multiplies the fp32 result of the row's dot product.
 *   Everything else as xshare_moe_forward (workspace from xshare_moe_workspace_bytes); shared
 *   experts are not taken here.
 */
xshare_status xshare_moe_forward_fp8(const uint16_t* x, const float* logits, int32_t T,
                                     int32_t d, int32_t f, const uint8_t* w1, const uint8_t* w3,
                                     const uint8_t* w2, const float* w1_scale,
                                     const float* w3_scale, const float* w2_scale,
                                     const xshare_route_params* params,
                                     const int32_t* req_offsets, const int32_t* host_offsets,
                                     int32_t R, const xshare_ep_layout* ep, uint16_t* y,
                                     uint8_t* sel_mask, int32_t* topk_ids, float* topk_w,
                                     xshare_stats* stats, void* ws, size_t ws_bytes,
                                     void* const* stage_events, hipStream_t stream);

/*
 * xshare_mx_scales_tile -- lays out MXFP4 block scales for the expert GEMMs (done once, when
 * the weights are loaded; not part of a layer call).  The GEMMs read one 16-row weight tile
 * over 256 inputs per load step: in the tiled layout that tile's scale bytes are one
 * contiguous 128-byte piece, read once, where the row-major layout scatters them over 16
 * rows (and the weight stream evicted those lines between steps).
 *
 *   scales  [n_mat, rows, k/32] uint8: E8M0 scales, one per block of 32 consecutive inputs
 *           of a row (row-major, as the OCP MX format lists them).
 *   tiled   [n_mat, rows/16, G, 16, 8] uint8 with G = ceil(k / 256):
 *           tiled[m][r / 16][c / 8][r % 16][c % 8] = scales[m][r][c]; bytes past a row's
 *           last block are 127 (scale 1) and never read.  Size:
 *           xshare_mx_scales_tiled_bytes(n_mat, rows, k).  Caller-owned device memory.
 *   rows a multiple of 16, k a multiple of 32 (XSHARE_EINVAL otherwise).  Asynchronous on
 *   `stream`; `scales` and `tiled` must not overlap.
 */
size_t xshare_mx_scales_tiled_bytes(int32_t n_mat, int32_t rows, int32_t k);
xshare_status xshare_mx_scales_tile(const uint8_t* scales, uint8_t* tiled, int32_t n_mat,
                                    int32_t rows, int32_t k, hipStream_t stream);

/*
 * xshare_moe_forward_mxfp4 -- xshare_moe_forward with MXFP4 routed-expert weights (OCP
 * Microscaling MXFP4: a quarter of the bytes of bf16 plus one scale byte per 32 weights;
 * the paper is silent on precision).
 *
 *   w1, w3    [N, f, d/2] uint8: FP4 E2M1 codes (1 sign, 2 exponent bits with bias 1, 1
 *             mantissa bit; values 0, 0.5, 1, 1.5, 2, 3, 4, 6 and their negatives), two per
 *             byte along the input index: element 2c in the low nibble of byte c.  16-byte
 *             aligned.
 *   w2        [N, d, f/2] uint8, same format.
 *   w1_scale, w3_scale  E8M0 scales of W1 and W3 ([N, f, d/32] row-major) in the tiled
 *             layout of xshare_mx_scales_tile (n_mat = N, rows = f, k = d); w2_scale those
 *             of W2 ([N, d, f/32]: rows = d, k = f).  One scale per block of 32 consecutive
 *             inputs of a row, value 2^(e - 127); the weight is decode(code) * 2^(e - 127).
 *             e = 255 (NaN) must not occur, and the decoded weights must lie in bf16's
 *             normal range (or be zero): the GPU turns each code and its scale into the
 *             exact bf16 weight before the bf16 MFMA.  16-byte aligned (XSHARE_EINVAL
 *             otherwise).
 *   d and f multiples of 32.  Everything else as xshare_moe_forward (workspace from
 *   xshare_moe_workspace_bytes); shared experts are not taken here.
 */
xshare_status xshare_moe_forward_mxfp4(const uint16_t* x, const float* logits, int32_t T,
                                       int32_t d, int32_t f, const uint8_t* w1,
                                       const uint8_t* w3, const uint8_t* w2,
                                       const uint8_t* w1_scale, const uint8_t* w3_scale,
                                       const uint8_t* w2_scale,
                                       const xshare_route_params* params,
                                       const int32_t* req_offsets, const int32_t* host_offsets,
                                       int32_t R, const xshare_ep_layout* ep, uint16_t* y,
                                       uint8_t* sel_mask, int32_t* topk_ids, float* topk_w,
                                       xshare_stats* stats, void* ws, size_t ws_bytes,
                                       void* const* stage_events, hipStream_t stream);

/*
 * xshare_moe_layer -- the whole MoE layer of Section 2.1 from the hidden states: router
 * logits h = W_g x (as xshare_router_logits), selection, the selected routed experts and
 * the shared experts, combine.
 *
 *   w_gate      [N, d] bf16 router weights (16-byte aligned).
 *   logits_out  nullable out [T, N] fp32: the logits the selection used (written by the
 *               router GEMM; bit-identical to xshare_router_logits on the same inputs).
 *   ws          at least xshare_layer_workspace_bytes.
 *   Other arguments as xshare_moe_forward; stage event 1 marks the end of router plus
 *   selection.
 */
xshare_status xshare_moe_layer(const uint16_t* x, const uint16_t* w_gate, int32_t T, int32_t d,
                               int32_t f, const uint16_t* w1, const uint16_t* w3,
                               const uint16_t* w2, const xshare_shared_experts* shared,
                               const xshare_route_params* params, const int32_t* req_offsets,
                               const int32_t* host_offsets, int32_t R,
                               const xshare_ep_layout* ep, uint16_t* y, float* logits_out,
                               uint8_t* sel_mask, int32_t* topk_ids, float* topk_w,
                               xshare_stats* stats, void* ws, size_t ws_bytes,
                               void* const* stage_events, hipStream_t stream);

/*
 * Uniform per-layer budgets for a global budget of K experts over L MoE layers (the uniform
 * allocation m_l = K / L of Section 3.2): m[l] = floor(K / L) + (l < K mod L ? 1 : 0), so
 * the budgets sum to exactly K and differ by at most one (when L divides K every layer gets
 * K / L).  Each m[l] is then a layer's XSHARE_BUDGET_TOTAL budget; a layer still selects at
 * least k experts, so the pass exceeds K when K / L < k (the ledger shows it).
 *   m   HOST [L] int32 output.   XSHARE_EINVAL if L < 1, K < 0 or m is NULL.
 * Host only: enqueues nothing.
 */
xshare_status xshare_layer_budgets(int32_t K, int32_t L, int32_t* m);

/*
 * xshare_probe_stream_read -- measurement only: a plain coalesced read of `bytes` bytes at
 * `buf` (16-byte aligned, a multiple of 16) by `blocks` workgroups of 256 threads, lanes
 * reading consecutive 16-byte pieces.  mode 0 / 1: the whole grid strides through the
 * buffer with 4 / 8 loads in flight per thread; mode 2 / 3: each workgroup reads its own
 * contiguous chunk, 4 / 8 loads in flight.  Timing it gives the HBM read rate a simple
 * kernel reaches on this GPU, the practical ceiling for the expert GEMMs' weight streams
 * (decode is bound by reading expert weights, Section 2.3).  `sink`: DEVICE uint32, written
 * at most once (it keeps the loads).  Asynchronous on `stream`; XSHARE_EINVAL for bad
 * arguments.
 */
xshare_status xshare_probe_stream_read(const void* buf, size_t bytes, int32_t blocks,
                                       int32_t mode, uint32_t* sink, hipStream_t stream);

/*
 * xshare_block_times -- measurement only: the block timeline of the expert GEMMs, from the
 * profiling build of this library (libxshare_timeline.so, compiled with XS_BLOCK_TIMES=1;
 * the product build returns XSHARE_EUNSUPPORTED and touches nothing).  That build stamps,
 * from the GPU's 100 MHz global clock, the start and end of every block of the last gate/up
 * and down launches, and the start and the end of each unit of every block of the last
 * persistent down launch; this call copies the stamps, asynchronously on `stream`, into
 * DEVICE uint64 arrays owned by the caller:
 *   gate_up     [2 * XSHARE_TIME_BLOCKS]: start, end of block b at 2b, 2b + 1, where
 *               b = (blockIdx.z * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x;
 *   down        [2 * XSHARE_TIME_BLOCKS]: the same for the down launch's grid;
 *   down_units  [XSHARE_TIME_SEQ_BLOCKS * XSHARE_TIME_SEQ_STRIDE]: block b of a persistent
 *               down launch at b * XSHARE_TIME_SEQ_STRIDE: its start, then its units' ends.
 * A launch overwrites only the entries of its own blocks (blocks past the array sizes are
 * not stamped), and blocks with no work stamp nothing; with `clear` nonzero the call zeroes
 * the stamps after copying them (hipMemsetAsync: a measurement call, not for capture in a
 * HIP graph).  XSHARE_EINVAL for a NULL pointer.
 */
#define XSHARE_TIME_BLOCKS 16384
#define XSHARE_TIME_SEQ_BLOCKS 1024
#define XSHARE_TIME_SEQ_STRIDE 33
xshare_status xshare_block_times(uint64_t* gate_up, uint64_t* down, uint64_t* down_units,
                                 int32_t clear, hipStream_t stream);

/* Static description of a status code (never NULL).                                      */
const char* xshare_status_string(int32_t status);

/* Library version, e.g. "0.1.0".                                                         */
const char* xshare_version(void);

#ifdef __cplusplus
}
#endif

#endif /* XSHARE_H */
