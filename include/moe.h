/*
 * moe.h — C ABI of the MI355X (gfx950) MoE-layer library (libmoe.so).
 *
 * The library runs one GPU's share of the DeepSeek-V3 Mixture-of-Experts layer
 * that the paper reproduces (App. M, "DeepSeek-V3 MoE Dispatch and Combine";
 * §4 Workloads; the host pipeline listing in App. F): gating and top-k
 * routing, dispatch of tokens to experts, the per-expert SwiGLU FFN
 * (GEMM1 gate/up projection, SwiGLU, GEMM2 down projection) and the weighted
 * combine. On one GPU the dispatch and combine all-to-alls of the paper become
 * an on-device permutation and its inverse. The paper does not define the
 * gate, scores, top-k rule or combine weights; the library implements the
 * public DeepSeek-V3 rule (sigmoid scores, selection bias, group-limited
 * top-k, normalised and scaled weights) and the Mixtral rule (softmax, top-k,
 * renormalised).
 *
 * Conventions for every call
 * --------------------------
 *  - Every pointer argument is a DEVICE pointer owned by the caller, except
 *    the config pointer and the debug-struct pointer (host memory). The library
 *    never allocates or frees device memory; scratch space is the caller's
 *    workspace `ws` of at least moe_workspace_size() bytes, passed with its
 *    size `ws_bytes`.
 *  - Calls validate their arguments synchronously, then enqueue kernels on the
 *    given stream(s) and return without synchronising. A non-zero return
 *    means nothing was enqueued (validation) or a launch failed (MOE_ERR_HIP);
 *    moe_last_error() then holds a message (per calling thread).
 *  - T = 0 is a valid no-op. No C++ exception crosses this interface.
 *  - Layouts are row-major and dense:
 *      x          [T][d]          activations, dtype
 *      w_router   [E][d]          router weight, one row per expert, dtype
 *      bias       [E]             fp32 selection bias (sigmoid routing only)
 *      w_gate     [E][I][d]       expert gate projections (GEMM1, gate half)
 *      w_up       [E][I][d]       expert up projections   (GEMM1, up half)
 *      w_down     [E][d][I]       expert down projections (GEMM2)
 *      ws_gate, ws_up [I_shared][d], ws_down [d][I_shared]  shared expert
 *    Every weight matrix is stored output-feature-major, so its reduction
 *    dimension is contiguous.
 *  - dtype MOE_BF16: activations and weights bf16, every product accumulated
 *    in fp32, the SwiGLU output and the expert outputs rounded to bf16 (round
 *    to nearest even). dtype MOE_F32: fp32 throughout.
 *  - Supported: 1 <= E <= 256, 1 <= k <= min(E, 16), d and I multiples of 64,
 *    n_shared in {0, 1}; larger or other shapes return MOE_ERR_UNSUPPORTED.
 *    The routed-expert weights are row-major unless cfg->weight_layout is
 *    MOE_LAYOUT_PACKED (see moe_pack_weights).
 *    Inputs must be finite.
 *  - Results are deterministic: two calls on the same inputs give the same
 *    bits, whatever the stream arrangement. (With packed weights the expert
 *    GEMMs hand out tiles to workgroups through atomic counters, but every
 *    output element is still computed in one fixed order.)
 *  - Calls that share one workspace must not overlap in time.
 *  - Calls enqueue kernels and (moe_layer with s_aux, moe_ep_expert_ffn)
 *    event records and waits only: no allocation, copy, memset or host
 *    synchronisation. A call (after one eager call of it on the device from
 *    the capturing thread, which sets up the kernels' attributes on that
 *    device and the thread's events)
 *    may therefore be captured in a HIP graph; each replay reads the
 *    buffers' contents at replay time (moe_layer's replays are tested to
 *    give the bits of eager calls).
 */
#ifndef MOE_H
#define MOE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MOE_OK = 0,
  MOE_ERR_INVALID_ARG = -1, /* NULL required pointer, T < 0, inconsistent config */
  MOE_ERR_UNSUPPORTED = -2, /* valid but outside the supported shapes/dtypes  */
  MOE_ERR_WORKSPACE = -3,   /* ws_bytes smaller than moe_workspace_size()     */
  MOE_ERR_HIP = -4          /* a HIP runtime call or kernel launch failed     */
} moe_status_t;

typedef enum { MOE_F32 = 0, MOE_BF16 = 1 } moe_dtype_t;

typedef enum {
  MOE_SCORE_SOFTMAX = 0, /* Mixtral: softmax scores, selection on the logit     */
  MOE_SCORE_SIGMOID = 1  /* DeepSeek-V3: sigmoid scores, selection on s + bias  */
} moe_score_t;

/* Layout of the expert weights passed to moe_expert_ffn, moe_shared_ffn and
 * moe_layer (routed and shared experts alike). */
typedef enum {
  MOE_LAYOUT_ROWMAJOR = 0, /* w_gate, w_up [E][I][d]; w_down [E][d][I]                       */
  MOE_LAYOUT_PACKED = 1    /* from moe_pack_weights: w_gate = packed gate+up, w_up = NULL,
                              w_down = packed down; bf16 only, I % 128 == 0, d % 256 == 0,
                              T*d and T*k*I below 2^31 elements                               */
} moe_layout_t;

/* Compression of the tokens the routed experts receive (App. F pipeline:
 * quantize before the dispatch exchange, dequantize before GEMM1). */
typedef enum {
  MOE_QUANT_NONE = 0, /* the routed experts see the bf16/fp32 tokens                */
  MOE_QUANT_INT8 = 1, /* int8 codes with one fp32 scale per token (moe_quantize);
                         bf16 and MOE_LAYOUT_PACKED only; the gate and the shared
                         expert, on the sending side, keep the original tokens       */
  MOE_QUANT_FP8 = 2   /* FP8 codes (OCP E4M3: 1 sign, 4 exponent bits with bias 7,
                         3 mantissa bits; largest value 448, 0x7F/0xFF NaN) with one
                         fp32 scale per token (Table 5's FP8 quantize); same rules   */
} moe_quant_t;

typedef struct {
  int32_t d;           /* hidden size                                         */
  int32_t E;           /* routed experts                                      */
  int32_t k;           /* experts selected per token                          */
  int32_t n_groups;    /* expert groups for the group limit (1 = no limit)    */
  int32_t topk_groups; /* groups kept per token                               */
  int32_t I;           /* routed-expert intermediate size                     */
  int32_t n_shared;    /* shared experts, 0 or 1                              */
  int32_t I_shared;    /* shared-expert intermediate size                     */
  int32_t score;       /* moe_score_t                                         */
  int32_t renorm;      /* 1: divide the selected scores by their sum          */
  float route_scale;   /* multiplies every weight (1.0 Mixtral, 2.5 DSV3)     */
  int32_t dtype;       /* moe_dtype_t                                         */
  int32_t weight_layout; /* moe_layout_t of the routed-expert weights          */
  int32_t token_quant;   /* moe_quant_t of the routed experts' input tokens    */
} moe_config_t;

/* Optional device buffers moe_layer writes its intermediates into (each may be
 * NULL; a NULL entry keeps that intermediate in the workspace). Sizes as in
 * moe_route/moe_dispatch/moe_expert_ffn/moe_shared_ffn. */
typedef struct {
  float* logits;          /* [T][E]   */
  int32_t* topk_idx;      /* [T][k]   */
  float* topk_w;          /* [T][k]   */
  int32_t* counts;        /* [E]      */
  int32_t* offsets;       /* [E+1]    */
  int32_t* sorted_token;  /* [T*k]    */
  int32_t* sorted_assign; /* [T*k]    */
  int32_t* inv_perm;      /* [T*k]    */
  void* y_perm;           /* [T*k][d] dtype */
  void* shared_out;       /* [T][d]   dtype (n_shared = 1 only) */
} moe_layer_debug_t;

/* Bytes of workspace any call below needs for this config and token count
 * (the maximum over the calls; 0 if the config is invalid). */
size_t moe_workspace_size(const moe_config_t* cfg, int32_t T);

/*
 * moe_route — gating and top-k routing (App. M: each token is routed to its
 * experts before the dispatch; selection rule as in the header comment).
 *  x, w_router : if x != NULL, logits = x · w_routerᵀ is computed (fp32
 *                accumulation) and written to `logits`; if x == NULL,
 *                `logits` is an input and w_router and ws are ignored.
 *  bias        : [E] fp32 added to the sigmoid scores for selection only;
 *                may be NULL (no bias); must be NULL for softmax routing.
 *  logits      : [T][E] fp32, required.
 *  topk_idx    : [T][k] int32 out, each row ordered by key descending, lower
 *                expert index first on ties.
 *  topk_w      : [T][k] fp32 out: selected scores (softmax probabilities or
 *                unbiased sigmoid), divided by their sum if cfg->renorm, times
 *                cfg->route_scale.
 *  ws          : workspace (required when x != NULL: the router GEMM may split
 *                its reduction into fp32 partial sums, which the routing
 *                kernel adds in a fixed order).
 * Keys, group scores and weights are evaluated in fp64 from the fp32 logits,
 * so the selection is a deterministic function of the logits' bits.
 */
int moe_route(const moe_config_t* cfg, int32_t T, const void* x, const void* w_router,
              const float* bias, float* logits, int32_t* topk_idx, float* topk_w, void* ws,
              size_t ws_bytes, hipStream_t stream);

/*
 * moe_dispatch — the single-GPU form of the dispatch all-to-all (App. F,
 * first exchange of the host pipeline; App. M: variable-size, unpadded
 * per-destination transfers). Assignment a = t*k + j sends token t to expert
 * topk_idx[t][j]; rows are grouped by expert, tokens ascending inside a group.
 *  counts        : [E] out, assignments per expert.
 *  offsets       : [E+1] out, exclusive prefix sum of counts (offsets[E] = T*k).
 *  sorted_token  : [T*k] out, token of every dispatched row.
 *  sorted_assign : [T*k] out or NULL, assignment of every row.
 *  inv_perm      : [T*k] out, row of every assignment.
 *  ws            : workspace (per-chunk expert masks and bases).
 * Every row of topk_idx is expected to hold k distinct experts in [0, E), as
 * moe_route writes them. An id outside [0, E) is skipped: its assignment gets
 * no row (its inv_perm entry is not written), offsets[E] counts only the
 * valid assignments, and rows past offsets[E] are not written. An expert
 * repeated within one row gives unspecified rows, but never an access out of
 * bounds.
 */
int moe_dispatch(const moe_config_t* cfg, int32_t T, const int32_t* topk_idx, int32_t* counts,
                 int32_t* offsets, int32_t* sorted_token, int32_t* sorted_assign,
                 int32_t* inv_perm, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * moe_dispatch_noalloc — moe_dispatch with no workspace argument, for callers
 * that cannot allocate device memory or pass a workspace: code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation.
 * Same arguments (minus ws, ws_bytes) and the same results as moe_dispatch.
 * Its per-chunk expert masks and bases live in a device array owned by the
 * library, one copy per GPU of 3 MiB, held until the process ends; the call
 * finds its address on its first use on each device and allocates nothing.
 * Limit: ceil(T / 64) * E <= 262144 (T <= 65536 tokens at E = 256); beyond it
 * the call returns MOE_ERR_UNSUPPORTED and enqueues nothing. Nothing in the
 * array needs to start at zero: a call writes every entry it reads. All calls
 * on one GPU share that array: calls ordered on one stream are safe, calls
 * that overlap in time on one GPU (several streams or threads) race and give
 * undefined results.
 */
int moe_dispatch_noalloc(const moe_config_t* cfg, int32_t T, const int32_t* topk_idx, int32_t* counts,
                         int32_t* offsets, int32_t* sorted_token, int32_t* sorted_assign, int32_t* inv_perm,
                         hipStream_t stream);

/*
 * moe_expert_ffn — the per-expert SwiGLU FFN over the dispatched rows
 * (App. M step 3 / App. F: GEMM1 gate+up, SwiGLU, GEMM2 down), as one grouped
 * GEMM pair: for every expert e and row r in [offsets[e], offsets[e+1]):
 *   h[r]      = silu(x[sorted_token[r]] · w_gate[e]ᵀ) * (x[sorted_token[r]] · w_up[e]ᵀ)
 *   y_perm[r] = h[r] · w_down[e]ᵀ
 * The row gather is fused into the GEMM's operand load. h lives in the
 * workspace (dtype, [T*k][I]); with packed weights so do the GEMMs' tile-queue
 * heads, which the call resets before its first GEMM.
 *  y_perm : [T*k][d] dtype out.
 */
int moe_expert_ffn(const moe_config_t* cfg, int32_t T, const void* x,
                   const int32_t* sorted_token, const int32_t* offsets, const void* w_gate,
                   const void* w_up, const void* w_down, void* y_perm, void* ws,
                   size_t ws_bytes, hipStream_t stream);

/*
 * moe_quantize — per-token quantization of the tokens (App. F pipeline,
 * the step before the dispatch exchange; App. M step (1); Table 5's FP8
 * quantize), selected by cfg->token_quant:
 *  MOE_QUANT_FP8: scale[t]    = max_c |x[t][c]| / 448                 (fp32)
 *                 codes[t][c] = E4M3 code of x[t][c] / scale[t], the fp32
 *                               quotient clamped to [-448, 448] and rounded
 *                               to the nearest value, ties to even;
 *  otherwise int8: scale[t]    = max_c |x[t][c]| / 127                 (fp32)
 *                 codes[t][c] = x[t][c] / scale[t] in fp32, rounded half to
 *                               even, clamped to [-127, 127].
 * A zero row: scale 0, codes 0 (code 0x80, E4M3 -0, marks a negative value
 * that rounds to zero).
 *  x : [T][d] bf16 (cfg->dtype must be MOE_BF16).
 *  codes : [T][d] bytes out (int8, or E4M3 bit patterns).   scales : [T] fp32 out.
 */
int moe_quantize(const moe_config_t* cfg, int32_t T, const void* x, int8_t* codes, float* scales,
                 hipStream_t stream);

/*
 * moe_expert_ffn_q8 — moe_expert_ffn on quantized tokens (App. M step (3):
 * dequantize + GEMM1 + SwiGLU + GEMM2): for every expert e and row r,
 *   t = sorted_token[r], h[r] = silu(s_t q_t · w_gate[e]ᵀ) * (s_t q_t · w_up[e]ᵀ),
 *   y_perm[r] = h[r] · w_down[e]ᵀ
 * with q_t the values of codes[t] (int8, or E4M3 when cfg->token_quant is
 * MOE_QUANT_FP8) and s_t = scales[t]. The dequantization is fused into
 * GEMM1: the gathered code rows are converted to bf16 (exactly) as they are
 * loaded, and each row's sums are multiplied by its scale before the SwiGLU.
 * Packed weights only (cfg->weight_layout == MOE_LAYOUT_PACKED, bf16).
 *  codes : [T][d] bytes, scales : [T] fp32 (from moe_quantize, same cfg).
 *  w_gate_up, w_down : packed weights from moe_pack_weights.
 *  y_perm : [T*k][d] bf16 out.
 */
int moe_expert_ffn_q8(const moe_config_t* cfg, int32_t T, const int8_t* codes, const float* scales,
                      const int32_t* sorted_token, const int32_t* offsets, const void* w_gate_up,
                      const void* w_down, void* y_perm, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * moe_shared_ffn — the shared expert: the same SwiGLU FFN, with intermediate
 * size cfg->I_shared, applied to all T tokens (dense, unweighted).
 *  ws_gate, ws_up, ws_down : row-major, or with MOE_LAYOUT_PACKED the output
 *        of moe_pack_weights for the shared expert alone (a config with E = 1
 *        and I = I_shared): ws_gate = packed gate+up, ws_up = NULL,
 *        ws_down = packed down.
 *  out : [T][d] dtype out. Requires cfg->n_shared == 1.
 */
int moe_shared_ffn(const moe_config_t* cfg, int32_t T, const void* x, const void* ws_gate,
                   const void* ws_up, const void* ws_down, void* out, void* ws,
                   size_t ws_bytes, hipStream_t stream);

/*
 * moe_combine — the single-GPU form of the combine all-to-all (App. F, second
 * exchange): a weighted gather back to token order,
 *   out[t] = sum_{j=0..k-1} topk_w[t][j] * y_perm[inv_perm[t*k+j]]  (+ shared_out[t])
 * with the slots summed in ascending j in fp32 and the shared expert added with
 * weight 1 when shared_out != NULL. No atomics: each output row is produced
 * by one workgroup.
 *  out : [T][d] dtype out.
 */
int moe_combine(const moe_config_t* cfg, int32_t T, const void* y_perm, const int32_t* inv_perm,
                const float* topk_w, const void* shared_out, void* out, hipStream_t stream);

/*
 * moe_layer — the whole layer: route, dispatch, expert FFN and combine on
 * s_main; the shared expert on s_aux, overlapping the routing and dispatch
 * (the single-GPU form of the paper's two-stream overlap, §4.3: dispatch on
 * one stream concurrent with expert compute on another, joined by an event).
 *  s_aux  : may be NULL or equal to s_main (then everything runs on s_main).
 *  ws_*   : shared-expert weights, required iff cfg->n_shared == 1, in the
 *           layout of cfg->weight_layout (see moe_shared_ffn). With packed
 *           weights and I_shared == I the shared expert is not run on s_aux:
 *           it is computed inside the routed expert GEMMs as one more group
 *           (its compute fills the matrix cores of the memory-bound routed
 *           work); the result is the same.
 *           With cfg->token_quant MOE_QUANT_INT8 or MOE_QUANT_FP8 the tokens are quantized
 *           first (moe_quantize, into the workspace) and the routed experts
 *           run on the codes (moe_expert_ffn_q8); the gate and the shared
 *           expert use x. With packed weights and I_shared == I the shared
 *           expert's GEMM1 then runs on its own on s_main and its GEMM2
 *           inside the routed GEMM2.
 *  out    : [T][d] dtype out.
 *  dbg    : NULL, or device buffers to receive intermediates (see above).
 * On return, s_main carries all the work (s_aux is joined into it).
 */
int moe_layer(const moe_config_t* cfg, int32_t T, const void* x, const void* w_router,
              const float* bias, const void* w_gate, const void* w_up, const void* w_down,
              const void* ws_gate, const void* ws_up, const void* ws_down, void* out, void* ws,
              size_t ws_bytes, hipStream_t s_main, hipStream_t s_aux, moe_layer_debug_t* dbg);

/*
 * moe_pack_weights — one-time conversion of the routed-expert weights into
 * the packed layout read by the weight-streaming expert GEMMs (a layout
 * choice of this library, not of the paper: it makes each K step of a
 * workgroup's weights one contiguous block already in matrix-core operand
 * order, so the memory-bound expert FFN streams the weights linearly).
 *  w_gate, w_up : [E][I][d] row-major bf16; gate_up_packed: 2*E*I*d bf16 out
 *                 (NULL: skipped).
 *  w_down       : [E][d][I] row-major bf16; down_packed: E*d*I bf16 out
 *                 (NULL: skipped).
 * cfg->weight_layout is ignored; requires bf16, I % 128 == 0, d % 256 == 0.
 * Packed layout per expert (8 bf16 per 16-byte chunk, k = s*64 + kk*16 +
 * 8*(lane >= 32) + 0..7):
 *  gate_up: [I/128][d/64 s][4 w][4 kk][2 j][64 lane][8], column
 *           t*128 + w*32 + lane%32 of w_gate (j = 0) or w_up (j = 1);
 *  down:    [d/256][I/64 s][4 w][4 kk][2 j][64 lane][8], output column
 *           t*256 + w*64 + j*32 + lane%32.
 */
int moe_pack_weights(const moe_config_t* cfg, const void* w_gate, const void* w_up, const void* w_down,
                     void* gate_up_packed, void* down_packed, hipStream_t stream);

/* ---- Receive side of expert parallelism (one GPU's share) --------------
 *
 * The paper's MoE workload (App. M; §4.3, Table 5) spreads the experts over
 * GPUs: the dispatch exchange brings each GPU the token rows routed to its
 * experts, its own tokens' rows ("self", available at once) and the peers'
 * ("remote", available once the exchange has delivered them). The calls
 * below run that receive side on one GPU, with the exchange's delivery of
 * the remote rows emulated by a copy whose rate is set by the workgroups it
 * may use (it runs on its own stream next to the expert GEMMs).
 *
 * Receive buffer: n_rows rows of d elements (cfg->dtype), one per (token,
 * local expert) assignment, grouped by local expert e in [0, cfg->E):
 *   rows [offsets[e], self_end[e])      self rows:   row of x_self
 *   rows [self_end[e], offsets[e + 1])  remote rows: row of x_peer
 * with row_token[r] the row's token in its source. offsets [E+1] and
 * self_end [E] are device int32 arrays, row_token [n_rows]. All three calls
 * need packed bf16 weights (moe_pack_weights, the E local experts) and
 * unquantized tokens; the workspace is moe_workspace_size(cfg,
 * ceil(n_rows / k)) bytes. Malformed offsets or indices are clamped
 * (unspecified rows, never an access out of bounds).
 */
typedef enum { MOE_EP_SELF = 0, MOE_EP_REMOTE = 1 } moe_ep_source_t;

/* moe_ep_plan — the receive buffer's layout for the local experts, global
 * experts [e_first, e_first + cfg->E), from this GPU's dispatch and the
 * peer's (moe_dispatch over the global experts: offsets [>= e_first+E+1],
 * sorted_token [assignments]): expert e's rows are this GPU's rows of that
 * expert then the peer's, each in its dispatch order (token ascending):
 *   offsets[e]  = (self_offsets[g] - self_offsets[e_first])
 *               + (peer_offsets[g] - peer_offsets[e_first]),  g = e_first + e
 *   self_end[e] = offsets[e] + self count of g
 *   row_token   : the tokens in that order.
 * Stands in for the exchange of per-expert counts between GPUs. Outputs:
 * offsets [E+1], self_end [E], row_token [capacity] (rows past the capacity
 * are not written). */
int moe_ep_plan(const moe_config_t* cfg, int32_t e_first, const int32_t* self_offsets, const int32_t* self_sorted_token,
                int32_t self_assignments, const int32_t* peer_offsets, const int32_t* peer_sorted_token,
                int32_t peer_assignments, int32_t* row_token, int32_t capacity, int32_t* offsets, int32_t* self_end,
                hipStream_t stream);

/* moe_ep_copy_rows — fills the rows of one source (moe_ep_source_t) of the
 * experts [e_begin, e_end): recv[r] = x_src[row_token[r]].
 *  x_src : [src_tokens][d]; recv : [n_rows][d].
 *  max_workgroups > 0 caps the copy's workgroups (the emulated link's rate;
 *  0: as many as fill the device). */
int moe_ep_copy_rows(const moe_config_t* cfg, int32_t source, int32_t n_rows, const void* x_src, int32_t src_tokens,
                     const int32_t* row_token, const int32_t* offsets, const int32_t* self_end, int32_t e_begin,
                     int32_t e_end, void* recv, int32_t max_workgroups, hipStream_t stream);

/* moe_expert_ffn_segments — moe_expert_ffn over row segments of a receive
 * buffer (App. M step 3), for experts e in [e_begin, e_end) and rows r in
 * [seg_begin[e], seg_end[e]) (seg_end NULL: [seg_begin[e], seg_begin[e+1]),
 * seg_begin then holding E+1 entries; index arrays need 4-byte alignment):
 *   h[r] = silu(x[r] · w_gate[e]ᵀ) * (x[r] · w_up[e]ᵀ),   y[r] = h[r] · w_down[e]ᵀ
 * x, y : [n_rows][d] (no gather; rows outside the segments are untouched).
 * max_workgroups > 0 caps the GEMMs' workgroups (leaving compute units to
 * kernels on other streams); 0: one per compute unit. */
int moe_expert_ffn_segments(const moe_config_t* cfg, int32_t n_rows, const void* x, const int32_t* seg_begin,
                            const int32_t* seg_end, int32_t e_begin, int32_t e_end, const void* w_gate_up,
                            const void* w_down, void* y, int32_t max_workgroups, void* ws, size_t ws_bytes,
                            hipStream_t stream);

/* Order of the receive side's work (§4.3: DeepEP's sequential phases vs the
 * two-stream pipeline the paper's search found). */
typedef enum {
  MOE_EP_SEQUENTIAL = 0,   /* all rows received, then one FFN over them */
  MOE_EP_SELF_REMOTE = 1,  /* the self rows' FFN while the remote rows arrive, then the
                              remote rows' FFN once all of them are in (the paper's split;
                              every expert's weights are streamed twice) */
  MOE_EP_EXPERT_CHUNKS = 2 /* the remote rows arrive by expert range; each range's FFN,
                              self and remote rows together, starts once its rows are in
                              (every expert's weights streamed once) */
} moe_ep_schedule_t;

typedef struct {
  int32_t schedule;        /* moe_ep_schedule_t                                        */
  int32_t chunks;          /* MOE_EP_EXPERT_CHUNKS: expert ranges, 1 .. min(16, E)     */
  int32_t link_workgroups; /* workgroups of the remote rows' copy (0: no cap)          */
  int32_t gemm_workgroups; /* workgroups of the GEMMs that run while rows still arrive
                              (0: one per compute unit)                                */
} moe_ep_options_t;

/* moe_ep_expert_ffn — the receive side in one call: the self rows copied
 * into recv on s_compute, the remote rows on s_link (the exchange), and the
 * FFN of every row into y on s_compute, ordered by opt->schedule; s_compute
 * waits for s_link's work before the call's last kernel, so everything is
 * complete when s_compute reaches the end of the call. s_link NULL (or equal
 * to s_compute): one stream. y[r] is the same for every schedule.
 *  x_self : [self_tokens][d]; x_peer : [peer_tokens][d];
 *  recv, y : [n_rows][d] out. */
int moe_ep_expert_ffn(const moe_config_t* cfg, const moe_ep_options_t* opt, int32_t n_rows, const void* x_self,
                      int32_t self_tokens, const void* x_peer, int32_t peer_tokens, const int32_t* row_token,
                      const int32_t* offsets, const int32_t* self_end, const void* w_gate_up, const void* w_down,
                      void* recv, void* y, void* ws, size_t ws_bytes, hipStream_t s_compute, hipStream_t s_link);

/* Static text for a moe_status_t. */
const char* moe_status_string(int status);
/* Message of the last failing call on this thread ("" if none). */
const char* moe_last_error(void);
/* Library version string. */
const char* moe_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MOE_H */
