/*
 * moe.h -- C ABI of the MI355X (gfx950) MoE-layer library (libmoe_mi355x.so): the forward
 * of one MoE layer and its backward.
 *
 * The library computes the forward pass of one Mixture-of-Experts layer on one
 * expert-parallel rank's share of the work: router logits, top-k gating, the
 * per-expert histogram and prefix scan of local (token, expert) pairs, the
 * permutation of token rows into expert-contiguous order, the grouped SwiGLU
 * expert MLP (plus an optional shared expert) and the gate-weighted combine.
 * These are the steps a generated MoE expert kernel performs in the paper's
 * kernel-generation design (Section 3.1, kernel sub-plan: permute before the
 * grouped GEMM, weighted combine after it; Section 4, kernel generation: the
 * monotone [E+1] row-offset array; Section 4, engine registration: the forward
 * composes the expert MLP's two GEMMs).  The training leg's backward of the expert MLP and
 * of the whole layer (moe_grouped_ffn_backward, moe_layer_backward) reuses the forward's
 * routing and permutation.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Pointers.  Every tensor argument is a DEVICE pointer owned by the caller.
 *    bf16 tensors are row-major, contiguous, 16-byte aligned; int32 / float
 *    arrays are contiguous and 4-byte aligned.  The library allocates no device
 *    memory on any call path; scratch space comes from the caller's workspace,
 *    whose size moe_workspace_size() returns (moe_permute_noalloc takes none: its
 *    scratch is a fixed device array of the library).
 *  - Streams.  `stream` is a hipStream_t passed as an opaque pointer (NULL = the
 *    legacy default stream).  Each call validates its arguments on the host; on
 *    success it enqueues its kernels on `stream` and returns without waiting.
 *    No call synchronises the device or reads device memory on the host: the
 *    number of local rows stays on the device.
 *  - Errors.  Calls return a moe_status_t.  On any status other than MOE_OK
 *    nothing was enqueued (except MOE_ERR_HIP, which reports a failed launch),
 *    and moe_last_error() returns a thread-local message naming the offending
 *    argument and its value.  There is no silent fallback: an unsupported shape
 *    is an error, never a slower path.
 *  - Limits.  d, F and F_shared are multiples of 8 (16-byte rows of bf16);
 *    1 <= E <= 1024; 1 <= top_k <= min(E, 16); T * top_k < 2^31; E_local <= 1024.
 *    T == 0 is a valid no-op.  Results for inputs holding Inf or NaN are
 *    unspecified.
 *  - Determinism.  Every output is bit-identical from run to run (no floating-
 *    point atomics), except moe_layer_forward with MOE_FUSE_COMBINE, whose expert
 *    rows are added into the token rows with float32 atomics in no fixed order.
 *
 * Layouts
 * -------
 *    x          [T, d]             bf16  token rows
 *    w_router   [E, d]             bf16  router weight, logits = x . w_router^T
 *    bias       [E]                f32   optional softmax-mode router bias (NULL = 0)
 *    topk_idx   [T, top_k]         i32   chosen GLOBAL expert ids, slot order = key descending
 *    topk_w     [T, top_k]         f32   gate of each slot
 *    counts     [E_local]          i32   local slots per local expert
 *    offsets    [E_local + 1]      i32   exclusive scan of counts (offsets[0] = 0)
 *    row_token  [cap]              i32   token of each expert-contiguous row (rows >= offsets[E_local] untouched)
 *    slot_row   [T, top_k]         i32   row of each slot, -1 when the expert is not local
 *    x_perm     [cap, d]           bf16  x_perm[r] = x[row_token[r]]
 *    w13        [E_local, 2F, d]   bf16  per local expert: rows [0,F) = W1 (gate), rows [F,2F) = W3 (up)
 *    w2         [E_local, d, F]    bf16  per local expert down projection
 *    y_perm     [cap, d]           bf16  expert MLP output of each row
 *    ws13/ws2   [2F_s, d] / [d, F_s]     shared expert (same packing), applied to every token with weight 1
 *    out        [T, d]             bf16
 *  with cap = T * min(top_k, E_local), the most local rows a batch can produce.
 *
 *  Masked-decode layout (shape->expert_capacity = C > 0; the equal-stride capacity
 *  offsets plus valid counts of the paper's kernel-generation section): cap = E_local * C,
 *  local expert e owns rows [e C, e C + min(counts[e], C)) and offsets[e] = e C; counts[e]
 *  stays the number of slots routed to e, of which the first C (ascending token) are kept
 *  and the others dropped (slot_row = -1, no routed contribution).  Every buffer size and
 *  every launch shape then depends on the shape only, not on the routing.
 */
#ifndef MOE_MI355X_H
#define MOE_MI355X_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MOE_ABI_VERSION 5

/* moe_shape_t.fusion: which of the paper's four kernel structures moe_layer_forward runs
 * (Section 4, kernel generation: fuse_gather folds the token permute into the first GEMM's
 * prologue, fuse_combine folds the weighted combine into the second GEMM's epilogue).
 * 0 = the library's choice (gather folded where its 32-bit row offsets reach all of x,
 * combine separate); otherwise MOE_FUSION_SET | any of MOE_FUSE_GATHER, MOE_FUSE_COMBINE. */
#define MOE_FUSION_SET 0x10
#define MOE_FUSE_GATHER 0x1
#define MOE_FUSE_COMBINE 0x2

typedef enum moe_status {
  MOE_OK = 0,
  MOE_ERR_INVALID_ARG = 1,  /* null / misaligned pointer, inconsistent shape field      */
  MOE_ERR_UNSUPPORTED = 2,  /* a valid request outside the kernels' stated limits        */
  MOE_ERR_WORKSPACE = 3,    /* ws_bytes smaller than moe_workspace_size() or ws == NULL  */
  MOE_ERR_HIP = 4           /* a HIP runtime call or kernel launch failed                */
} moe_status_t;

typedef enum moe_gate {
  MOE_GATE_SOFTMAX = 0,     /* key = logit + bias; gate = softmax over the chosen keys (renormalize=1)
                               or over all experts (renormalize=0); times routed_scale   */
  MOE_GATE_SIGMOID = 1      /* key = sigmoid(logit); gate = key / sum of chosen keys (renormalize=1)
                               or key (renormalize=0); times routed_scale; no bias        */
} moe_gate_t;

/* Which call a workspace is sized for (moe_workspace_size). */
typedef enum moe_ws_kind {
  MOE_WS_ROUTE = 0,
  MOE_WS_PERMUTE = 1,
  MOE_WS_FFN = 2,
  MOE_WS_LAYER = 3,
  MOE_WS_FFN_BWD = 4,
  MOE_WS_LAYER_BWD = 5
} moe_ws_kind_t;

/* Named regions inside a MOE_WS_LAYER workspace (moe_workspace_offset). */
typedef enum moe_ws_region {
  MOE_REGION_TOPK_IDX = 0,   /* i32 [T, top_k]   */
  MOE_REGION_TOPK_W = 1,     /* f32 [T, top_k]   */
  MOE_REGION_COUNTS = 2,     /* i32 [E_local]    */
  MOE_REGION_OFFSETS = 3,    /* i32 [E_local+1]  */
  MOE_REGION_ROW_TOKEN = 4,  /* i32 [cap]        */
  MOE_REGION_SLOT_ROW = 5,   /* i32 [T, top_k]   */
  MOE_REGION_X_PERM = 6,     /* bf16 [cap, d]; written by moe_layer_forward only when the gather is
                                not folded (the up-projection otherwise reads x through row_token) */
  MOE_REGION_Y_PERM = 7,     /* bf16 [cap, d]; not written when the combine is folded */
  MOE_REGION_SHARED_Y = 8,   /* bf16 [T, d] (only when F_shared > 0; not written when the
                                combine is folded) */
  MOE_REGION_COUNT_ = 9
} moe_ws_region_t;

/* Shape and gating of one MoE layer on one expert-parallel rank (passed by pointer).
 * The rank holds experts [e_begin, e_begin + E_local) of the E routed experts; a slot
 * routed elsewhere is dropped from this rank's compute.  With n_group > 1 the E
 * experts form n_group contiguous groups, a group scores the sum of its two largest
 * keys, and only experts of the topk_group best groups are eligible.  Top-k ties go
 * to the lower expert (group) index. */
typedef struct moe_shape {
  int64_t T;            /* tokens                                       */
  int32_t d;            /* hidden size                                  */
  int32_t E;            /* routed experts of the whole layer            */
  int32_t top_k;        /* experts per token                            */
  int32_t e_begin;      /* first local expert                           */
  int32_t E_local;      /* local experts                                */
  int32_t F;            /* routed expert FFN width                      */
  int32_t F_shared;     /* shared expert FFN width, 0 = none            */
  int32_t gate;         /* moe_gate_t                                   */
  int32_t n_group;      /* expert groups, 1 = no group limit            */
  int32_t topk_group;   /* groups kept per token when n_group > 1       */
  int32_t renormalize;  /* 0 or 1                                       */
  float routed_scale;   /* multiplies every routed gate                 */
  int32_t expert_capacity; /* 0: rows of all local experts packed by the monotone
                              [E_local+1] offsets; C > 0: masked-decode layout, expert e
                              owns the equal-stride segment [e C, e C + C) and keeps its
                              first C slots (ascending token), later slots are dropped */
  int32_t fusion;       /* moe_layer_forward's kernel structure: 0 or MOE_FUSION_SET | flags
                           (see MOE_FUSE_GATHER / MOE_FUSE_COMBINE); ignored by the other calls */
} moe_shape_t;

/* Library ABI version (MOE_ABI_VERSION of the build). */
int moe_abi_version(void);

/* Static description of a status code. */
const char* moe_status_string(int status);

/* Message of the last failed call on this thread ("" if none). */
const char* moe_last_error(void);

/* Bytes of caller workspace the call `kind` needs for `shape` (0 for an invalid shape;
 * moe_last_error() then says why).  Always a multiple of 256. */
size_t moe_workspace_size(const moe_shape_t* shape, int kind);

/* Byte offset of a named region inside a MOE_WS_LAYER workspace, so a caller can read
 * the routing, permutation and intermediate rows of the last moe_layer_forward on that
 * workspace.  Returns (size_t)-1 for an invalid shape or region. */
size_t moe_workspace_offset(const moe_shape_t* shape, int region);

/* Router logits, gating and top-k (steps 1-5 of the layer).  The paper states routing only in
 * prose (Section 2, background: each token is routed to a small subset of experts); the gate
 * formulas are the readings fixed by moe_gate_t and the group limit by n_group / topk_group.
 * Writes topk_idx and topk_w; when keys_out [T, E] f32 is not NULL it also receives
 * the float32 key every decision was taken on (softmax: logit + bias; sigmoid: the
 * sigmoid score), so a checker can replay the decision in the same precision.
 * Logits accumulate bf16 products in float32.  ws: MOE_WS_ROUTE bytes. */
int moe_route(const moe_shape_t* shape, const void* x, const void* w_router, const float* bias,
              int32_t* topk_idx, float* topk_w, float* keys_out,
              void* ws, size_t ws_bytes, void* stream);

/* Histogram, prefix scan and permutation (steps 6-8; Section 3.1, kernel spec: the token permute
 * ahead of the grouped GEMM; Section 4, kernel generation: each expert's rows are the segment of
 * a monotone [E+1] offset array, or the valid prefix of an equal-stride capacity segment).
 * From topk_idx, keeps the slots whose expert lies in [e_begin, e_begin + E_local),
 * writes counts and the monotone offsets (expert e owns rows [offsets[e], offsets[e+1])),
 * orders the rows of one expert by ascending token (a stable counting sort), writes
 * row_token and slot_row, and gathers x_perm[r] = x[row_token[r]] (bit-exact copy).
 * Masked-decode layout (expert_capacity C > 0): offsets[e] = e C, rows e C + rank for the
 * slots ranked below C, the others dropped; row_token and x_perm are written for the kept
 * rows only.
 * ws: MOE_WS_PERMUTE bytes. */
int moe_permute(const moe_shape_t* shape, const int32_t* topk_idx, const void* x,
                int32_t* counts, int32_t* offsets, int32_t* row_token, int32_t* slot_row,
                void* x_perm, void* ws, size_t ws_bytes, void* stream);

/* moe_permute without a workspace argument, for callers that cannot allocate device memory
 * (code under HIP graph capture, serving loops that forbid allocation).  Same arguments,
 * results and layouts as moe_permute; its scratch (per-chunk counts and bases,
 * moe_workspace_size(shape, MOE_WS_PERMUTE) bytes, about 12 * ceil(T / 64) * E_local) lives in
 * a fixed 1 MiB device array owned by the library, one per device, kept until the process
 * ends.  Larger requests (e.g. E_local = 128 with T > 43000) return MOE_ERR_UNSUPPORTED.  The call
 * allocates nothing; the first call on a device looks up the array's address there.
 * Every call on one GPU shares that GPU's array: calls that may overlap on one GPU (other
 * streams, other threads) race on it and must be ordered by the caller. */
int moe_permute_noalloc(const moe_shape_t* shape, const int32_t* topk_idx, const void* x,
                        int32_t* counts, int32_t* offsets, int32_t* row_token, int32_t* slot_row,
                        void* x_perm, void* stream);

/* Grouped SwiGLU expert MLP (step 9; Section 4, engine registration: the forward composes the
 * expert MLP's two GEMMs; Section 4, kernel generation: one kernel body reads each expert's rows
 * through the offset array, or through capacity offsets plus valid counts in masked decode).
 * For every local expert e and every row r in
 * [offsets[e], offsets[e+1]):  y_perm[r] = W2_e (silu(W1_e x_perm[r]) * (W3_e x_perm[r])).
 * The activation is rounded to bf16 before the second GEMM; accumulation is float32.
 * `offsets` is a device array of E_local + 1 entries (e.g. from moe_permute) and must
 * satisfy 0 = offsets[0] <= ... <= offsets[E_local] <= cap (entries are clamped to [0, cap]).
 * Masked-decode layout (expert_capacity C > 0): `offsets` is instead the device array of the
 * E_local per-expert counts (e.g. moe_permute's `counts`); expert e runs rows
 * [e C, e C + min(counts[e], C)).  The shared expert is this call with E_local = 1,
 * F = F_shared, expert_capacity = 0 and offsets = {0, T} over x.
 * ws: MOE_WS_FFN bytes. */
int moe_grouped_ffn(const moe_shape_t* shape, const void* x_perm, const int32_t* offsets,
                    const void* w13, const void* w2, void* y_perm,
                    void* ws, size_t ws_bytes, void* stream);

/* Backward of the grouped SwiGLU expert MLP (the paper's training leg, Section 4, engine
 * registration: the backward composes the expert kernels' dual GEMMs in transposed layout
 * for the activation gradient and per-expert products for the weight gradients).
 * For the rows r of local expert e (the segments of moe_grouped_ffn, either layout) and
 * the gradient dy_perm of its output rows:
 *   H = x W1^T, U = x W3^T (recomputed), dA = dy W2,
 *   dH = dA * U * silu'(H), dU = dA * silu(H),
 *   dx_perm[r] = [dH dU] w13                  (bf16 [cap, d]; rows outside every segment are
 *                                              not written)
 *   dw13[e] = [dH dU]^T x,  dw2[e] = dy^T (silu(H) * U)   (bf16 [E_local, 2F, d] / [E_local, d, F];
 *                                              an expert without rows gets zeros)
 * fp32 accumulation; dA, [dH dU] and the recomputed activation are rounded to bf16 once
 * each (workspace), as are the results.  The activation-gradient GEMMs read w2 and w13 in
 * their stored layout (the transposed operand of the forward), the weight-gradient GEMMs
 * read the row-major activations as transposed operands (no transposed copies are made).
 * ws: MOE_WS_FFN_BWD bytes. */
int moe_grouped_ffn_backward(const moe_shape_t* shape, const void* x_perm, const int32_t* offsets,
                             const void* w13, const void* w2, const void* dy_perm,
                             void* dx_perm, void* dw13, void* dw2,
                             void* ws, size_t ws_bytes, void* stream);

/* Backward of the whole layer (the paper's training leg, Section 4, engine registration: the
 * forward composes the expert kernels' two GEMMs, the backward their dual GEMMs), for the
 * output gradient dout [T, d] of the moe_layer_forward call that left its state in fwd_ws
 * (same shape and inputs; the choice of experts is that forward's and carries no gradient):
 *   dgate[t, j] = <dout[t], y_perm[row(t, j)]>            (local slots; 0 for the others)
 *   expert rows: dy_perm[row(t, j)] = topk_w[t, j] dout[t], then the expert-MLP backward
 *                (as moe_grouped_ffn_backward) -> dx rows, dw13, dw2
 *   shared expert: its MLP backward for dout on every token -> dx rows, dws13, dws2
 *   gates -> router logits: d key from dgate by the derivative of the gate formula
 *                (shape->gate / renormalize / routed_scale; see moe_gate_t), times
 *                k (1 - k) for sigmoid keys; the keys are recomputed bit-identically from
 *                the forward's float32 logit partials
 *   router: dx += dlogits w_router,  dw_router = dlogits^T x
 *   dx[t] = bf16( sum of the token's expert-row gradients (slot order) + shared + router ),
 *           float32 accumulation, one rounding.
 * A router bias is a constant (no gradient).  Outputs: dx [T, d], dw_router [E, d],
 * dw13 [E_local, 2F, d], dw2 [E_local, d, F], dws13 [2F_s, d], dws2 [d, F_s] (the last two
 * only when F_shared > 0), all bf16 and written in full (an expert without rows gets zeros).
 * Rounded to bf16 once each on the way: dlogits, the expert rows' output gradients, and the
 * expert-MLP backward's intermediates (as moe_grouped_ffn_backward).
 * fwd_ws / fwd_ws_bytes: the MOE_WS_LAYER workspace of that forward, whose routing,
 * permutation, logit partials and expert output rows are read; the forward must not have
 * folded the combine (MOE_FUSE_COMBINE leaves no expert output rows: MOE_ERR_UNSUPPORTED).
 * The backward writes the forward's MOE_REGION_X_PERM region (the expert-ordered token rows).
 * Also requires E % 8 == 0 (the router GEMMs reduce over, and produce, rows of E values).
 * ws: MOE_WS_LAYER_BWD bytes (gradient rows and GEMM intermediates). */
int moe_layer_backward(const moe_shape_t* shape, const void* x, const void* w_router, const float* bias,
                       const void* w13, const void* w2, const void* ws13, const void* ws2,
                       const void* dout, void* fwd_ws, size_t fwd_ws_bytes,
                       void* dx, void* dw_router, void* dw13, void* dw2, void* dws13, void* dws2,
                       void* ws, size_t ws_bytes, void* stream);

/* Gate-weighted combine (steps 10-11; Section 3.1, kernel spec: the weighted combine after the
 * grouped GEMM, or folded into its epilogue as fuse_combine):
 *   out[t] = bf16( sum over slots j with slot_row[t,j] >= 0 of topk_w[t,j] * y_perm[slot_row[t,j]]
 *                  + shared_y[t] )
 * accumulated in float32 in slot order, the shared row (NULL = none) added last, one
 * round-to-nearest-even to bf16.  A token with no local slot gets shared_y[t] (or 0). */
int moe_combine(const moe_shape_t* shape, const void* y_perm, const int32_t* slot_row,
                const float* topk_w, const void* shared_y, void* out, void* stream);

/* The whole layer: route -> permute -> grouped_ffn (+ shared expert) -> combine.
 * Kernel structure (shape->fusion; Section 3.1 kernel sub-plan, Section 4 kernel generation):
 *  - gather folded (MOE_FUSE_GATHER, and the default when T * d * 2 < 2^32): the
 *    up-projection reads its token rows from x through row_token, x_perm is not written;
 *    unfolded, the permutation copies the rows into x_perm first.  Results are identical.
 *    An explicit MOE_FUSE_GATHER with T * d * 2 >= 2^32 is MOE_ERR_UNSUPPORTED.
 *  - combine folded (MOE_FUSE_COMBINE): the down-projection's epilogue adds
 *    topk_w * (expert row, float32) into a float32 [T, d] accumulator with atomics (the shared
 *    expert's rows with weight 1), and one pass rounds it to bf16; y_perm and shared_y are not
 *    written.  The expert rows are not rounded to bf16 first, and the order of the additions
 *    is not fixed, so results may differ from run to run in the last bf16 bit.
 *  Default (fusion = 0): gather folded where allowed, combine separate.
 * ws13 / ws2 are required when F_shared > 0 and ignored otherwise.
 * ws: MOE_WS_LAYER bytes; its named regions hold the intermediates afterwards. */
int moe_layer_forward(const moe_shape_t* shape, const void* x, const void* w_router, const float* bias,
                      const void* w13, const void* w2, const void* ws13, const void* ws2,
                      void* out, void* ws, size_t ws_bytes, void* stream);

/* Steps of moe_layer_forward, in launch order (moe_layer_forward_traced). */
typedef enum moe_step {
  MOE_STEP_ROUTER_GEMM = 0,   /* router logits (grouped GEMM, one group, f32 out)   */
  MOE_STEP_GATE = 1,          /* gating + top-k                                     */
  MOE_STEP_HISTOGRAM = 2,     /* per-chunk histogram + scan over chunks             */
  MOE_STEP_PERMUTE = 3,       /* offsets, stable ranks (+ row copy when not folded) */
  MOE_STEP_FFN_UP = 4,        /* routed experts: W1/W3 GEMM + SwiGLU                */
  MOE_STEP_FFN_DOWN = 5,      /* routed experts: W2 GEMM                            */
  MOE_STEP_SHARED_UP = 6,     /* shared expert: W1/W3 GEMM + SwiGLU (if F_shared)   */
  MOE_STEP_SHARED_DOWN = 7,   /* shared expert: W2 GEMM (if F_shared)               */
  /* when F_shared == F the shared expert runs inside the two routed launches (steps 4 and 5
     then cover both and steps 6 and 7 are empty) */
  MOE_STEP_COMBINE = 8,       /* gate-weighted combine                              */
  MOE_STEP_COUNT_ = 9
} moe_step_t;

/* moe_layer_forward with per-step timing for profilers and benchmarks: `events` holds
 * MOE_STEP_COUNT_ + 1 hipEvent_t (as opaque pointers) created by the caller; events[i]
 * is recorded on `stream` right before step i is enqueued and events[MOE_STEP_COUNT_]
 * after the last step (a step that does not run gets its event recorded all the same,
 * so its interval is empty; with T == 0 every event is recorded, back to back).  A NULL
 * entry is not recorded: each recorded event adds a few microseconds of GPU time to the
 * step, so a caller timing only some steps passes only their boundaries.
 * events == NULL behaves exactly like moe_layer_forward. */
int moe_layer_forward_traced(const moe_shape_t* shape, const void* x, const void* w_router, const float* bias,
                             const void* w13, const void* w2, const void* ws13, const void* ws2,
                             void* out, void* ws, size_t ws_bytes, void* const* events, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* MOE_MI355X_H */
