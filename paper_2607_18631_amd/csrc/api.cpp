// C ABI of the MoE-layer forward: argument validation, workspace layout, kernel dispatch.
// Every entry point validates on the host before touching the GPU, so an invalid call
// returns its status without any HIP call; a valid call only enqueues work on `stream`.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>

#include "../../include/moe.h"
#include "kernels.hpp"

namespace {

thread_local std::string g_err;

int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return status;
}

int ok() {
  g_err.clear();
  return MOE_OK;
}

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// rows of the expert-ordered buffers: every local slot (offsets layout) or E_local equal
// segments of expert_capacity rows (masked-decode layout)
int64_t capacity(const moe_shape_t* s) {
  if (s->expert_capacity > 0) return (int64_t)s->E_local * s->expert_capacity;
  return s->T * (int64_t)(s->top_k < s->E_local ? s->top_k : s->E_local);
}

// Expected rows per local expert of a layer call (tile-shape choice only; the real counts stay
// on the device): T * top_k / E under uniform routing, at most the expert capacity in the masked
// layout.  The standalone grouped-FFN entry points take their capacity / E_local instead (their
// rows fill the capacity they are given, e.g. the shared expert as one group of T rows).
int64_t expected_rows(const moe_shape_t* s) {
  int64_t r = std::max<int64_t>(1, s->T * s->top_k / std::max(1, s->E));
  if (s->expert_capacity > 0) r = std::min<int64_t>(r, s->expert_capacity);
  return r;
}

int check_shape(const moe_shape_t* s) {
  if (!s) return fail(MOE_ERR_INVALID_ARG, "shape is NULL");
  if (s->T < 0) return fail(MOE_ERR_INVALID_ARG, "T (%lld) < 0", (long long)s->T);
  if (s->d <= 0) return fail(MOE_ERR_INVALID_ARG, "d (%d) <= 0", s->d);
  if (s->d % 8) return fail(MOE_ERR_UNSUPPORTED, "d (%d) %% 8 != 0 (rows must be 16-byte bf16 vectors)", s->d);
  if (s->E < 1 || s->E > 1024) return fail(MOE_ERR_UNSUPPORTED, "E (%d) outside [1, 1024]", s->E);
  if (s->top_k < 1 || s->top_k > 16 || s->top_k > s->E)
    return fail(MOE_ERR_UNSUPPORTED, "top_k (%d) outside [1, min(E=%d, 16)]", s->top_k, s->E);
  if (s->T * (int64_t)s->top_k >= (int64_t(1) << 31))
    return fail(MOE_ERR_UNSUPPORTED, "T * top_k (%lld) >= 2^31", (long long)(s->T * s->top_k));
  if (s->e_begin < 0 || s->E_local < 1 || (int64_t)s->e_begin + s->E_local > s->E)
    return fail(MOE_ERR_INVALID_ARG, "local slice [e_begin=%d, e_begin+E_local=%d) not inside [0, E=%d)",
                s->e_begin, s->e_begin + s->E_local, s->E);
  if (s->F <= 0) return fail(MOE_ERR_INVALID_ARG, "F (%d) <= 0", s->F);
  if (s->F % 8) return fail(MOE_ERR_UNSUPPORTED, "F (%d) %% 8 != 0", s->F);
  if (s->F_shared < 0) return fail(MOE_ERR_INVALID_ARG, "F_shared (%d) < 0", s->F_shared);
  if (s->F_shared % 8) return fail(MOE_ERR_UNSUPPORTED, "F_shared (%d) %% 8 != 0", s->F_shared);
  if (s->gate != MOE_GATE_SOFTMAX && s->gate != MOE_GATE_SIGMOID)
    return fail(MOE_ERR_UNSUPPORTED, "gate (%d) is neither MOE_GATE_SOFTMAX nor MOE_GATE_SIGMOID", s->gate);
  if (s->n_group < 1) return fail(MOE_ERR_INVALID_ARG, "n_group (%d) < 1", s->n_group);
  if (s->E % s->n_group) return fail(MOE_ERR_INVALID_ARG, "E (%d) %% n_group (%d) != 0", s->E, s->n_group);
  if (s->n_group > 1) {
    if (s->n_group > 64) return fail(MOE_ERR_UNSUPPORTED, "n_group (%d) > 64", s->n_group);
    if (s->E / s->n_group < 2)
      return fail(MOE_ERR_INVALID_ARG, "group size E/n_group (%d) < 2: a group scores its two largest keys",
                  s->E / s->n_group);
    if (s->topk_group < 1 || s->topk_group > s->n_group)
      return fail(MOE_ERR_INVALID_ARG, "topk_group (%d) outside [1, n_group=%d]", s->topk_group, s->n_group);
    if ((int64_t)s->topk_group * (s->E / s->n_group) < s->top_k)
      return fail(MOE_ERR_INVALID_ARG, "topk_group * group size (%d) < top_k (%d)",
                  s->topk_group * (s->E / s->n_group), s->top_k);
  }
  if (s->renormalize != 0 && s->renormalize != 1)
    return fail(MOE_ERR_INVALID_ARG, "renormalize (%d) is not 0 or 1", s->renormalize);
  if (!std::isfinite(s->routed_scale)) return fail(MOE_ERR_INVALID_ARG, "routed_scale is not finite");
  if (s->expert_capacity < 0) return fail(MOE_ERR_INVALID_ARG, "expert_capacity (%d) < 0", s->expert_capacity);
  if ((int64_t)s->E_local * s->expert_capacity >= (int64_t(1) << 31))
    return fail(MOE_ERR_UNSUPPORTED, "E_local * expert_capacity (%lld) >= 2^31",
                (long long)((int64_t)s->E_local * s->expert_capacity));
  if (s->fusion != 0 && (!(s->fusion & MOE_FUSION_SET) ||
                         (s->fusion & ~(MOE_FUSION_SET | MOE_FUSE_GATHER | MOE_FUSE_COMBINE))))
    return fail(MOE_ERR_INVALID_ARG, "fusion (0x%x) is neither 0 nor MOE_FUSION_SET | MOE_FUSE_* flags", s->fusion);
  return MOE_OK;
}

// the up-projection reads token rows through row_token (per-lane 32-bit offsets into x)
bool gather_fits(const moe_shape_t* s) { return s->T * (int64_t)s->d * 2 < (int64_t(1) << 32); }
bool fuse_gather(const moe_shape_t* s) {
  return s->fusion == 0 ? gather_fits(s) : (s->fusion & MOE_FUSE_GATHER) != 0;
}
bool fuse_combine(const moe_shape_t* s) { return (s->fusion & MOE_FUSE_COMBINE) != 0;
}

int check_ptr(const void* p, size_t align, const char* name) {
  if (!p) return fail(MOE_ERR_INVALID_ARG, "%s is NULL", name);
  if (reinterpret_cast<uintptr_t>(p) % align)
    return fail(MOE_ERR_INVALID_ARG, "%s (%p) is not %zu-byte aligned", name, p, align);
  return MOE_OK;
}

#define CHECK(expr)          \
  do {                       \
    int _st = (expr);        \
    if (_st != MOE_OK) return _st; \
  } while (0)

// ---- workspace layouts ----
// router logits: one [T, E] fp32 partial per K chunk of the logits GEMM
size_t ws_route(const moe_shape_t* s) {
  return align_up((size_t)moe::logits_splits(s->T, s->E, s->d) * s->T * s->E * sizeof(float));
}
size_t ws_permute(const moe_shape_t* s) { return moe::permute_ws(s->T, s->E_local).bytes; }
size_t ws_ffn(const moe_shape_t* s) { return align_up((size_t)capacity(s) * s->F * sizeof(uint16_t)); }
// backward: dA [cap, F], [dH dU] [cap, 2F], recomputed activation [cap, F] (bf16)
size_t ws_ffn_bwd(const moe_shape_t* s) { return 4 * ws_ffn(s); }

struct LayerLayout {
  size_t region[MOE_REGION_COUNT_];
  size_t logits, perm_ws, act, act_s;
  size_t acc32, row_weight;   // combine folded into the down-projection only
  size_t total;
};

LayerLayout layer_layout(const moe_shape_t* s) {
  LayerLayout L{};
  const size_t T = (size_t)s->T, k = (size_t)s->top_k, cap = (size_t)capacity(s), d = (size_t)s->d;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += align_up(bytes);
    return o;
  };
  L.region[MOE_REGION_TOPK_IDX] = take(T * k * 4);
  L.region[MOE_REGION_TOPK_W] = take(T * k * 4);
  L.region[MOE_REGION_COUNTS] = take((size_t)s->E_local * 4);
  L.region[MOE_REGION_OFFSETS] = take(((size_t)s->E_local + 1) * 4);
  L.region[MOE_REGION_ROW_TOKEN] = take(cap * 4);
  L.region[MOE_REGION_SLOT_ROW] = take(T * k * 4);
  L.region[MOE_REGION_X_PERM] = take(cap * d * 2);
  L.region[MOE_REGION_Y_PERM] = take(cap * d * 2);
  L.region[MOE_REGION_SHARED_Y] = take(s->F_shared > 0 ? T * d * 2 : 0);
  L.logits = take(ws_route(s));
  L.perm_ws = take(ws_permute(s));
  L.act = take(ws_ffn(s));
  L.act_s = take(s->F_shared > 0 ? T * (size_t)s->F_shared * 2 : 0);
  L.acc32 = take(fuse_combine(s) ? T * d * 4 : 0);
  L.row_weight = take(fuse_combine(s) ? cap * 4 : 0);
  L.total = off;
  return L;
}

// Layer backward: gate gradients, logit gradients, the expert rows' output and input
// gradients, the shared expert's and the router's input gradients, and the expert-MLP
// backward's intermediates (routed and shared run one after the other on the same scratch).
struct LayerBwdLayout {
  size_t seg, segk, dgate, dlogits, dy_perm, dx_perm, dx_shared, dx_router, wr_parts, scratch;
  size_t total;
};

// K split of the router weight gradient dw_router = dlogits^T x (E x d outputs reduced over T
// tokens): at most one (chunk, m-tile, n-tile) tile per compute unit of the chip, chunks of at
// least 256 tokens, at most 16 chunks; float32 partials summed in chunk order.
constexpr int kWrSplitMax = 16;
int router_wgrad_splits(int64_t T, int E, int d) {
  const int64_t tiles = ((E + 255) / 256) * (int64_t)((d + 255) / 256);
  int64_t s = 256 / tiles;
  s = std::min<int64_t>(s, kWrSplitMax);
  s = std::min<int64_t>(s, std::max<int64_t>(1, T / 256));
  return (int)std::max<int64_t>(s, 1);
}
int64_t router_wgrad_chunk(int64_t T, int E, int d) {
  const int s = router_wgrad_splits(T, E, d);
  return std::max<int64_t>(1, (T + s - 1) / s);
}

LayerBwdLayout layer_bwd_layout(const moe_shape_t* s) {
  LayerBwdLayout L{};
  const size_t T = (size_t)s->T, k = (size_t)s->top_k, cap = (size_t)capacity(s), d = (size_t)s->d;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += align_up(bytes);
    return o;
  };
  L.seg = take(2 * sizeof(int32_t));
  L.segk = take((kWrSplitMax + 1) * sizeof(int32_t));
  L.dgate = take(T * k * 4);
  L.dlogits = take(T * (size_t)s->E * 2);
  L.dy_perm = take(cap * d * 2);
  L.dx_perm = take(cap * d * 2);
  L.dx_shared = take(s->F_shared > 0 ? T * d * 2 : 0);
  L.dx_router = take(T * d * 2);
  L.wr_parts = take((size_t)router_wgrad_splits(s->T, s->E, s->d) * s->E * d * 4);
  // ffn_backward takes four planes of align_up(rows * F * 2) bytes
  L.scratch = take(std::max(4 * align_up(cap * (size_t)s->F * 2), 4 * align_up(T * (size_t)s->F_shared * 2)));
  L.total = off;
  return L;
}

size_t ws_need(const moe_shape_t* s, int kind) {
  switch (kind) {
    case MOE_WS_ROUTE: return ws_route(s);
    case MOE_WS_PERMUTE: return ws_permute(s);
    case MOE_WS_FFN: return ws_ffn(s);
    case MOE_WS_LAYER: return layer_layout(s).total;
    case MOE_WS_FFN_BWD: return ws_ffn_bwd(s);
    case MOE_WS_LAYER_BWD: return layer_bwd_layout(s).total;
    default: return 0;
  }
}

int check_ws(const moe_shape_t* s, int kind, const void* ws, size_t ws_bytes) {
  const size_t need = ws_need(s, kind);
  if (need == 0) return MOE_OK;
  if (!ws) return fail(MOE_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if (reinterpret_cast<uintptr_t>(ws) % kAlign)
    return fail(MOE_ERR_INVALID_ARG, "workspace (%p) is not %zu-byte aligned", ws, kAlign);
  if (ws_bytes < need) return fail(MOE_ERR_WORKSPACE, "ws_bytes (%zu) < required (%zu)", ws_bytes, need);
  return MOE_OK;
}

int hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return MOE_OK;
  return fail(MOE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }
template <class T>
inline T* at(void* base, size_t off) { return reinterpret_cast<T*>(static_cast<char*>(base) + off); }

// ---- dispatch (arguments already validated) ----
using Marker = int (*)(int step);
thread_local void* const* g_events = nullptr;
thread_local hipStream_t g_event_stream = nullptr;
int mark_event(int step) {
  if (!g_events[step]) return MOE_OK;                     // not asked for
  return hip_status(hipEventRecord(static_cast<hipEvent_t>(g_events[step]), g_event_stream), "hipEventRecord");
}

int mark_permute() { return mark_event(MOE_STEP_PERMUTE); }

int do_route(const moe_shape_t* s, const void* x, const void* w_router, const float* bias, int32_t* topk_idx,
             float* topk_w, float* keys_out, float* logits, hipStream_t st, Marker mark = nullptr) {
  moe::GemmProblem g{};
  g.X = static_cast<const moe::bf16_t*>(x);
  g.ldx = s->d;
  g.offsets = nullptr;
  g.groups = 1;
  g.rows_single = s->T;
  g.max_rows = s->T;
  g.W = static_cast<const moe::bf16_t*>(w_router);
  g.w_group_stride = 0;
  g.N = s->E;
  g.K = s->d;
  g.Y = logits;
  g.ldy = s->E;
  g.epi = moe::EPI_F32;
  const int splits = moe::logits_splits(s->T, s->E, s->d);
  g.ksplit = splits;
  g.y_split_stride = s->T * (int64_t)s->E;
  CHECK(hip_status(moe::launch_grouped_gemm(g, st), "router logits launch"));
  if (mark) CHECK(mark(MOE_STEP_GATE));
  moe::GateProblem q{};
  q.logits = logits;
  q.nsplit = splits;
  q.split_stride = s->T * (int64_t)s->E;
  q.bias = bias;
  q.T = s->T;
  q.E = s->E;
  q.top_k = s->top_k;
  q.gate = s->gate;
  q.n_group = s->n_group;
  q.topk_group = s->topk_group;
  q.group_size = s->E / s->n_group;
  q.renormalize = s->renormalize;
  q.routed_scale = s->routed_scale;
  q.topk_idx = topk_idx;
  q.topk_w = topk_w;
  q.keys_out = keys_out;
  return hip_status(moe::launch_gate(q, st), "gating launch");
}

int do_permute(const moe_shape_t* s, const int32_t* topk_idx, const void* x, int32_t* counts, int32_t* offsets,
               int32_t* row_token, int32_t* slot_row, void* x_perm, void* ws, hipStream_t st,
               Marker mark = nullptr, const float* topk_w = nullptr, float* row_weight = nullptr) {
  moe::PermuteProblem p{};
  p.topk_idx = topk_idx;
  p.x = static_cast<const moe::bf16_t*>(x);
  p.T = s->T;
  p.d = s->d;
  p.top_k = s->top_k;
  p.e_begin = s->e_begin;
  p.E_local = s->E_local;
  p.counts = counts;
  p.offsets = offsets;
  p.row_token = row_token;
  p.slot_row = slot_row;
  p.x_perm = static_cast<moe::bf16_t*>(x_perm);
  p.cap = capacity(s);
  p.expert_capacity = s->expert_capacity;
  p.topk_w = topk_w;
  p.row_weight = row_weight;
  const moe::PermuteWs pw = moe::permute_ws(s->T, s->E_local);
  p.super_count = at<int32_t>(ws, pw.super_count);
  p.super_base = at<int32_t>(ws, pw.super_base);
  p.totals = at<int32_t>(ws, pw.totals);
  p.chunk_mask = at<uint64_t>(ws, pw.chunk_mask);
  p.chunk_base = at<int32_t>(ws, pw.chunk_base);
  return hip_status(moe::launch_permute(p, st, mark ? mark_permute : nullptr),
                    "permute launch");
}

// Shared expert run inside the routed launches (an extra GEMM group on its own operands).
struct SharedOperands {
  const void* x = nullptr;    // [T, d]
  const void* w13 = nullptr;  // [2F, d]
  const void* w2 = nullptr;   // [d, F]
  void* act = nullptr;        // [T, F]
  void* y = nullptr;          // [T, d]
  int64_t T = 0;
};

// `offsets`: the monotone [groups + 1] row offsets, or with seg_stride > 0 the [groups]
// row counts of equal segments of seg_stride rows (masked-decode layout).
//
// Gathered rows for the up-projection: row r of the grouped part is token row_index[r] of X
// (X has x_rows rows); row_index == nullptr means X is already in expert order.
struct Gather {
  const int32_t* row_index = nullptr;
  int64_t x_rows = 0;
};

// The combine folded into the down-projection: rows are added, times their gate, into the
// float32 token rows acc [rows, d] (token[r] / weight[r] of the grouped rows; null = the row
// itself / 1; the shared expert's rows always the row itself with weight 1).
struct Scatter {
  float* acc = nullptr;
  const int32_t* token = nullptr;
  const float* weight = nullptr;
  int64_t rows = 0;
};

int do_ffn(const void* X, const int32_t* offsets, int groups, int64_t rows, const void* w13, const void* w2,
           int d, int F, void* act, void* y, hipStream_t st, Marker mark = nullptr, int down_step = 0,
           const SharedOperands* sh = nullptr, Gather gather = Gather{}, int64_t rows_hint = 0,
           int seg_stride = 0, Scatter scatter = Scatter{}) {
  moe::GemmProblem up{};
  up.seg_stride = seg_stride;
  up.rows_hint = rows_hint > 0 ? rows_hint : (groups > 0 ? (rows + groups - 1) / groups : rows);
  up.X = static_cast<const moe::bf16_t*>(X);
  up.row_index = gather.row_index;
  up.x_rows = gather.x_rows;
  up.ldx = d;
  up.offsets = offsets;
  up.groups = groups;
  up.rows_single = rows;
  up.max_rows = rows;
  up.W = static_cast<const moe::bf16_t*>(w13);
  up.w_group_stride = (int64_t)2 * F * d;
  up.N = F;
  up.K = d;
  up.Y = act;
  up.ldy = F;
  up.epi = moe::EPI_SWIGLU;
  if (sh) {
    up.X2 = static_cast<const moe::bf16_t*>(sh->x);
    up.W2 = static_cast<const moe::bf16_t*>(sh->w13);
    up.Y2 = sh->act;
    up.rows2 = (int32_t)sh->T;
  }
  CHECK(hip_status(moe::launch_grouped_gemm(up, st), "expert up-projection launch"));
  if (mark) CHECK(mark(down_step));
  moe::GemmProblem dn = up;
  dn.row_index = nullptr;
  dn.x_rows = 0;
  dn.X = static_cast<const moe::bf16_t*>(act);
  dn.ldx = F;
  dn.W = static_cast<const moe::bf16_t*>(w2);
  dn.w_group_stride = (int64_t)d * F;
  dn.N = d;
  dn.K = F;
  dn.Y = y;
  dn.ldy = d;
  dn.epi = moe::EPI_BF16;
  if (sh) {
    dn.X2 = static_cast<const moe::bf16_t*>(sh->act);
    dn.W2 = static_cast<const moe::bf16_t*>(sh->w2);
    dn.Y2 = sh->y;
    dn.rows2 = (int32_t)sh->T;
  }
  if (scatter.acc) {
    dn.epi = moe::EPI_SCATTER;
    dn.Y = scatter.acc;
    if (sh) dn.Y2 = scatter.acc;
    dn.scatter_token = scatter.token;
    dn.scatter_weight = scatter.weight;
    dn.scatter_rows = scatter.rows;
  }
  return hip_status(moe::launch_grouped_gemm(dn, st), "expert down-projection launch");
}

int do_combine(const moe_shape_t* s, const void* y_perm, const int32_t* slot_row, const float* topk_w,
               const void* shared_y, void* out, hipStream_t st) {
  moe::CombineProblem c{};
  c.y_perm = static_cast<const moe::bf16_t*>(y_perm);
  c.slot_row = slot_row;
  c.topk_w = topk_w;
  c.shared_y = static_cast<const moe::bf16_t*>(shared_y);
  c.out = static_cast<moe::bf16_t*>(out);
  c.T = s->T;
  c.cap = capacity(s);
  c.d = s->d;
  c.top_k = s->top_k;
  return hip_status(moe::launch_combine(c, st), "combine launch");
}

// Expert-MLP backward (arguments validated): dA = dY W2, the up-projection recomputed with
// the SwiGLU-backward epilogue, dX = [dH dU] w13, dW2 = dY^T A, dW13 = [dH dU]^T X.
// Group g owns rows [offsets[g], offsets[g+1]) of x / dy / dx (or, with seg_stride > 0, the
// first min(offsets[g], seg_stride) rows of [g seg_stride, (g+1) seg_stride)); `rows` bounds
// them; scratch holds 4 rows x F bf16 values (dA, activation, [dH dU]).
struct FfnBwd {
  const void* x = nullptr;
  const int32_t* offsets = nullptr;
  int groups = 0;
  int64_t rows = 0, rows_hint = 0;
  int seg_stride = 0, d = 0, F = 0;
  bool any_rows = true;       // false: no token rows (only the weight gradients, all zero)
  const void *w13 = nullptr, *w2 = nullptr, *dy = nullptr;
  void *dx = nullptr, *dw13 = nullptr, *dw2 = nullptr, *scratch = nullptr;
};

int ffn_backward(const FfnBwd& a, hipStream_t st) {
  const int d = a.d, F = a.F;
  const size_t plane = align_up((size_t)a.rows * F * sizeof(uint16_t));
  auto* da = at<moe::bf16_t>(a.scratch, 0);
  auto* act = at<moe::bf16_t>(a.scratch, plane);
  auto* dhu = at<moe::bf16_t>(a.scratch, 2 * plane);
  moe::GemmBwdProblem g{};
  g.offsets = a.offsets;
  g.groups = a.groups;
  g.seg_stride = a.seg_stride;
  g.max_rows = a.rows;
  g.rows_hint = a.rows_hint;
  // dA = dY W2 (W2 [d][F] read as the transposed operand)
  g.mode = moe::BWD_ROWS;
  g.x_mn = false;
  g.w_mn = true;
  g.X = static_cast<const moe::bf16_t*>(a.dy);
  g.ldx = d;
  g.W = static_cast<const moe::bf16_t*>(a.w2);
  g.ldw = F;
  g.w_group_stride = (int64_t)d * F;
  g.N = F;
  g.K = d;
  g.Y = da;
  g.ldy = F;
  if (a.any_rows) CHECK(hip_status(moe::launch_gemm_bwd(g, st), "dA launch"));
  // recompute H, U; dH, dU and the activation from dA
  moe::GemmProblem up{};
  up.X = static_cast<const moe::bf16_t*>(a.x);
  up.ldx = d;
  up.offsets = a.offsets;
  up.groups = a.groups;
  up.rows_single = a.rows;
  up.max_rows = a.rows;
  up.seg_stride = a.seg_stride;
  up.rows_hint = a.rows_hint;
  up.W = static_cast<const moe::bf16_t*>(a.w13);
  up.w_group_stride = (int64_t)2 * F * d;
  up.N = F;
  up.K = d;
  up.Y = dhu;
  up.ldy = 2 * (int64_t)F;
  up.epi = moe::EPI_SWIGLU_BWD;
  up.dact = da;
  up.act_out = act;
  if (a.any_rows) CHECK(hip_status(moe::launch_grouped_gemm(up, st), "SwiGLU backward launch"));
  // dX = [dH dU] w13 (w13 [2F][d] read as the transposed operand)
  g.X = dhu;
  g.ldx = 2 * F;
  g.W = static_cast<const moe::bf16_t*>(a.w13);
  g.ldw = d;
  g.w_group_stride = (int64_t)2 * F * d;
  g.N = d;
  g.K = 2 * F;
  g.Y = static_cast<moe::bf16_t*>(a.dx);
  g.ldy = d;
  if (a.any_rows) CHECK(hip_status(moe::launch_gemm_bwd(g, st), "dX launch"));
  // weight gradients: reductions over each expert's rows (also with no tokens: then every
  // segment is empty and the launches write zeros)
  moe::GemmBwdProblem w = g;
  w.mode = moe::BWD_KSEG;
  w.x_mn = w.w_mn = true;
  w.w_group_stride = 0;
  // dW2[e] = dY^T A: [d, F]
  w.X = static_cast<const moe::bf16_t*>(a.dy);
  w.ldx = d;
  w.W = act;
  w.ldw = F;
  w.M = d;
  w.N = F;
  w.Y = static_cast<moe::bf16_t*>(a.dw2);
  w.ldy = F;
  w.y_group_stride = (int64_t)d * F;
  CHECK(hip_status(moe::launch_gemm_bwd(w, st), "dW2 launch"));
  // dW13[e] = [dH dU]^T X: [2F, d]
  w.X = dhu;
  w.ldx = 2 * F;
  w.W = static_cast<const moe::bf16_t*>(a.x);
  w.ldw = d;
  w.M = 2 * F;
  w.N = d;
  w.Y = static_cast<moe::bf16_t*>(a.dw13);
  w.ldy = d;
  w.y_group_stride = (int64_t)2 * F * d;
  return hip_status(moe::launch_gemm_bwd(w, st), "dW13 launch");
}

int do_ffn_backward(const moe_shape_t* s, const void* x_perm, const int32_t* offsets, const void* w13,
                    const void* w2, const void* dy, void* dx, void* dw13, void* dw2, void* ws, hipStream_t st) {
  FfnBwd a;
  a.x = x_perm;
  a.offsets = offsets;
  a.groups = s->E_local;
  a.rows = capacity(s);
  a.any_rows = s->T > 0;
  a.rows_hint = std::max<int64_t>(1, capacity(s) / s->E_local);
  a.seg_stride = s->expert_capacity;
  a.d = s->d;
  a.F = s->F;
  a.w13 = w13;
  a.w2 = w2;
  a.dy = dy;
  a.dx = dx;
  a.dw13 = dw13;
  a.dw2 = dw2;
  a.scratch = ws;
  return ffn_backward(a, st);
}

}  // namespace

extern "C" {

int moe_abi_version(void) { return MOE_ABI_VERSION; }

const char* moe_status_string(int status) {
  switch (status) {
    case MOE_OK: return "MOE_OK";
    case MOE_ERR_INVALID_ARG: return "MOE_ERR_INVALID_ARG: an argument is NULL, misaligned or inconsistent";
    case MOE_ERR_UNSUPPORTED: return "MOE_ERR_UNSUPPORTED: the request is outside the kernels' limits";
    case MOE_ERR_WORKSPACE: return "MOE_ERR_WORKSPACE: the workspace is missing or too small";
    case MOE_ERR_HIP: return "MOE_ERR_HIP: a HIP call or kernel launch failed";
    default: return "unknown moe_status_t";
  }
}

const char* moe_last_error(void) { return g_err.c_str(); }

size_t moe_workspace_size(const moe_shape_t* shape, int kind) {
  if (check_shape(shape) != MOE_OK) return 0;
  if (kind < MOE_WS_ROUTE || kind > MOE_WS_LAYER_BWD) {
    fail(MOE_ERR_INVALID_ARG, "workspace kind (%d) unknown", kind);
    return 0;
  }
  size_t n = ws_need(shape, kind);
  return n ? n : kAlign;
}

size_t moe_workspace_offset(const moe_shape_t* shape, int region) {
  if (check_shape(shape) != MOE_OK) return (size_t)-1;
  if (region < 0 || region >= MOE_REGION_COUNT_) {
    fail(MOE_ERR_INVALID_ARG, "region (%d) unknown", region);
    return (size_t)-1;
  }
  return layer_layout(shape).region[region];
}

int moe_route(const moe_shape_t* shape, const void* x, const void* w_router, const float* bias, int32_t* topk_idx,
              float* topk_w, float* keys_out, void* ws, size_t ws_bytes, void* stream) {
  CHECK(check_shape(shape));
  if (bias && shape->gate != MOE_GATE_SOFTMAX)
    return fail(MOE_ERR_UNSUPPORTED, "a router bias is only defined for softmax gating");
  if (shape->T == 0) return ok();
  CHECK(check_ptr(x, 16, "x"));
  CHECK(check_ptr(w_router, 16, "w_router"));
  if (bias) CHECK(check_ptr(bias, 4, "bias"));
  CHECK(check_ptr(topk_idx, 4, "topk_idx"));
  CHECK(check_ptr(topk_w, 4, "topk_w"));
  if (keys_out) CHECK(check_ptr(keys_out, 4, "keys_out"));
  CHECK(check_ws(shape, MOE_WS_ROUTE, ws, ws_bytes));
  CHECK(do_route(shape, x, w_router, bias, topk_idx, topk_w, keys_out, static_cast<float*>(ws), as_stream(stream)));
  return ok();
}

int moe_permute(const moe_shape_t* shape, const int32_t* topk_idx, const void* x, int32_t* counts, int32_t* offsets,
                int32_t* row_token, int32_t* slot_row, void* x_perm, void* ws, size_t ws_bytes, void* stream) {
  CHECK(check_shape(shape));
  if (shape->T == 0) return ok();
  CHECK(check_ptr(topk_idx, 4, "topk_idx"));
  CHECK(check_ptr(x, 16, "x"));
  CHECK(check_ptr(counts, 4, "counts"));
  CHECK(check_ptr(offsets, 4, "offsets"));
  CHECK(check_ptr(row_token, 4, "row_token"));
  CHECK(check_ptr(slot_row, 4, "slot_row"));
  CHECK(check_ptr(x_perm, 16, "x_perm"));
  CHECK(check_ws(shape, MOE_WS_PERMUTE, ws, ws_bytes));
  CHECK(do_permute(shape, topk_idx, x, counts, offsets, row_token, slot_row, x_perm, ws, as_stream(stream)));
  return ok();
}

int moe_permute_noalloc(const moe_shape_t* shape, const int32_t* topk_idx, const void* x, int32_t* counts,
                        int32_t* offsets, int32_t* row_token, int32_t* slot_row, void* x_perm, void* stream) {
  CHECK(check_shape(shape));
  const size_t need = ws_permute(shape);
  if (need > moe::kPermuteScratchBytes)
    return fail(MOE_ERR_UNSUPPORTED,
                "moe_permute_noalloc needs %zu bytes of scratch for T=%lld, E_local=%d; its fixed scratch holds %zu",
                need, (long long)shape->T, shape->E_local, moe::kPermuteScratchBytes);
  if (shape->T == 0) return ok();
  CHECK(check_ptr(topk_idx, 4, "topk_idx"));
  CHECK(check_ptr(x, 16, "x"));
  CHECK(check_ptr(counts, 4, "counts"));
  CHECK(check_ptr(offsets, 4, "offsets"));
  CHECK(check_ptr(row_token, 4, "row_token"));
  CHECK(check_ptr(slot_row, 4, "slot_row"));
  CHECK(check_ptr(x_perm, 16, "x_perm"));
  void* scratch = nullptr;
  CHECK(hip_status(moe::permute_scratch(&scratch), "scratch address lookup (hipGetSymbolAddress)"));
  CHECK(do_permute(shape, topk_idx, x, counts, offsets, row_token, slot_row, x_perm, scratch, as_stream(stream)));
  return ok();
}

int moe_grouped_ffn(const moe_shape_t* shape, const void* x_perm, const int32_t* offsets, const void* w13,
                    const void* w2, void* y_perm, void* ws, size_t ws_bytes, void* stream) {
  CHECK(check_shape(shape));
  if (shape->E_local > moe::kMaxGroups)
    return fail(MOE_ERR_UNSUPPORTED, "E_local (%d) > %d", shape->E_local, moe::kMaxGroups);
  if (shape->T == 0) return ok();
  CHECK(check_ptr(x_perm, 16, "x_perm"));
  CHECK(check_ptr(offsets, 4, "offsets"));
  CHECK(check_ptr(w13, 16, "w13"));
  CHECK(check_ptr(w2, 16, "w2"));
  CHECK(check_ptr(y_perm, 16, "y_perm"));
  CHECK(check_ws(shape, MOE_WS_FFN, ws, ws_bytes));
  CHECK(do_ffn(x_perm, offsets, shape->E_local, capacity(shape), w13, w2, shape->d, shape->F, ws, y_perm,
               as_stream(stream), nullptr, 0, nullptr, Gather{}, 0, shape->expert_capacity));
  return ok();
}

int moe_grouped_ffn_backward(const moe_shape_t* shape, const void* x_perm, const int32_t* offsets,
                             const void* w13, const void* w2, const void* dy_perm, void* dx_perm, void* dw13,
                             void* dw2, void* ws, size_t ws_bytes, void* stream) {
  CHECK(check_shape(shape));
  if (shape->E_local > moe::kMaxGroups)
    return fail(MOE_ERR_UNSUPPORTED, "E_local (%d) > %d", shape->E_local, moe::kMaxGroups);
  CHECK(check_ptr(dw13, 16, "dw13"));
  CHECK(check_ptr(dw2, 16, "dw2"));
  CHECK(check_ptr(offsets, 4, "offsets"));
  CHECK(check_ws(shape, MOE_WS_FFN_BWD, ws, ws_bytes));
  if (shape->T > 0) {
    CHECK(check_ptr(x_perm, 16, "x_perm"));
    CHECK(check_ptr(w13, 16, "w13"));
    CHECK(check_ptr(w2, 16, "w2"));
    CHECK(check_ptr(dy_perm, 16, "dy_perm"));
    CHECK(check_ptr(dx_perm, 16, "dx_perm"));
  }
  CHECK(do_ffn_backward(shape, x_perm, offsets, w13, w2, dy_perm, dx_perm, dw13, dw2, ws, as_stream(stream)));
  return ok();
}

int moe_layer_backward(const moe_shape_t* shape, const void* x, const void* w_router, const float* bias,
                       const void* w13, const void* w2, const void* ws13, const void* ws2, const void* dout,
                       void* fwd_ws, size_t fwd_ws_bytes, void* dx, void* dw_router, void* dw13, void* dw2,
                       void* dws13, void* dws2, void* ws, size_t ws_bytes, void* stream) {
  CHECK(check_shape(shape));
  const moe_shape_t* s = shape;
  if (s->E_local > moe::kMaxGroups) return fail(MOE_ERR_UNSUPPORTED, "E_local (%d) > %d", s->E_local, moe::kMaxGroups);
  if (bias && s->gate != MOE_GATE_SOFTMAX)
    return fail(MOE_ERR_UNSUPPORTED, "a router bias is only defined for softmax gating");
  if (fuse_combine(s))
    return fail(MOE_ERR_UNSUPPORTED,
                "the forward folded the combine (MOE_FUSE_COMBINE): it leaves no expert output rows for the gate "
                "gradients");
  if (s->E % 8)
    return fail(MOE_ERR_UNSUPPORTED, "E (%d) %% 8 != 0 (the router backward GEMMs take rows of E values)", s->E);
  CHECK(check_ptr(dw_router, 16, "dw_router"));
  CHECK(check_ptr(dw13, 16, "dw13"));
  CHECK(check_ptr(dw2, 16, "dw2"));
  if (s->F_shared > 0) {
    CHECK(check_ptr(dws13, 16, "dws13"));
    CHECK(check_ptr(dws2, 16, "dws2"));
  }
  hipStream_t st = as_stream(stream);
  const int64_t T = s->T;
  const int d = s->d, E = s->E, F = s->F, Fs = s->F_shared;
  if (T == 0) {
    // no tokens: every weight gradient is zero (bf16 zero = all-zero bits)
    auto zero = [&](void* p, int64_t elems, const char* what) {
      return hip_status(moe::launch_zero_f32(static_cast<float*>(p), elems / 2, st), what);
    };
    CHECK(zero(dw_router, (int64_t)E * d, "dw_router clear launch"));
    CHECK(zero(dw13, (int64_t)s->E_local * 2 * F * d, "dw13 clear launch"));
    CHECK(zero(dw2, (int64_t)s->E_local * d * F, "dw2 clear launch"));
    if (Fs > 0) {
      CHECK(zero(dws13, (int64_t)2 * Fs * d, "dws13 clear launch"));
      CHECK(zero(dws2, (int64_t)d * Fs, "dws2 clear launch"));
    }
    return ok();
  }
  CHECK(check_ptr(x, 16, "x"));
  CHECK(check_ptr(w_router, 16, "w_router"));
  if (bias) CHECK(check_ptr(bias, 4, "bias"));
  CHECK(check_ptr(w13, 16, "w13"));
  CHECK(check_ptr(w2, 16, "w2"));
  if (Fs > 0) {
    CHECK(check_ptr(ws13, 16, "ws13"));
    CHECK(check_ptr(ws2, 16, "ws2"));
  }
  CHECK(check_ptr(dout, 16, "dout"));
  CHECK(check_ptr(dx, 16, "dx"));
  CHECK(check_ws(s, MOE_WS_LAYER, fwd_ws, fwd_ws_bytes));
  CHECK(check_ws(s, MOE_WS_LAYER_BWD, ws, ws_bytes));

  const LayerLayout F0 = layer_layout(s);
  const LayerBwdLayout B = layer_bwd_layout(s);
  const int32_t* topk_idx = at<int32_t>(fwd_ws, F0.region[MOE_REGION_TOPK_IDX]);
  const float* topk_w = at<float>(fwd_ws, F0.region[MOE_REGION_TOPK_W]);
  const int32_t* counts = at<int32_t>(fwd_ws, F0.region[MOE_REGION_COUNTS]);
  const int32_t* offsets = at<int32_t>(fwd_ws, F0.region[MOE_REGION_OFFSETS]);
  const int32_t* slot_row = at<int32_t>(fwd_ws, F0.region[MOE_REGION_SLOT_ROW]);
  auto* x_perm = at<moe::bf16_t>(fwd_ws, F0.region[MOE_REGION_X_PERM]);
  const auto* y_perm = at<moe::bf16_t>(fwd_ws, F0.region[MOE_REGION_Y_PERM]);
  int32_t* seg = at<int32_t>(ws, B.seg);
  float* dgate = at<float>(ws, B.dgate);
  auto* dlogits = at<moe::bf16_t>(ws, B.dlogits);
  auto* dy_perm = at<moe::bf16_t>(ws, B.dy_perm);
  auto* dx_perm = at<moe::bf16_t>(ws, B.dx_perm);
  auto* dx_shared = Fs > 0 ? at<moe::bf16_t>(ws, B.dx_shared) : nullptr;
  auto* dx_router = at<moe::bf16_t>(ws, B.dx_router);
  void* scratch = at<void>(ws, B.scratch);
  const int64_t cap = capacity(s);
  const int C = s->expert_capacity;

  // combine backward: gate gradients and the expert rows' output gradients
  moe::CombineBwdProblem cb{};
  cb.dout = static_cast<const moe::bf16_t*>(dout);
  cb.y_perm = y_perm;
  cb.slot_row = slot_row;
  cb.topk_w = topk_w;
  cb.dgate = dgate;
  cb.dy_perm = dy_perm;
  cb.T = T;
  cb.cap = cap;
  cb.d = d;
  cb.top_k = s->top_k;
  CHECK(hip_status(moe::launch_combine_bwd(cb, st), "combine backward launch"));
  // gates -> logits (keys recomputed from the forward's partials); also the {0, T} segment
  moe::GateBwdProblem gb{};
  gb.logits = at<float>(fwd_ws, F0.logits);
  gb.nsplit = moe::logits_splits(T, E, d);
  gb.split_stride = T * (int64_t)E;
  gb.bias = bias;
  gb.topk_idx = topk_idx;
  gb.dgate = dgate;
  gb.T = T;
  gb.E = E;
  gb.top_k = s->top_k;
  gb.gate = s->gate;
  gb.renormalize = s->renormalize;
  gb.routed_scale = s->routed_scale;
  gb.dlogits = dlogits;
  gb.seg = seg;
  const int wr_splits = router_wgrad_splits(T, E, d);
  const int64_t wr_chunk = router_wgrad_chunk(T, E, d);
  // chunks actually covering [0, T) (the last ones may be empty when T is small)
  const int wr_groups = (int)std::min<int64_t>(wr_splits, (T + wr_chunk - 1) / wr_chunk);
  gb.segk = at<int32_t>(ws, B.segk);
  gb.nsegk = wr_groups;
  gb.segk_rows = wr_chunk;
  CHECK(hip_status(moe::launch_gate_bwd(gb, st), "gate backward launch"));
  // expert-ordered token rows (the forward may have read them straight from x)
  moe::PermuteProblem pp{};
  pp.x = static_cast<const moe::bf16_t*>(x);
  pp.T = T;
  pp.d = d;
  pp.top_k = s->top_k;
  pp.slot_row = const_cast<int32_t*>(slot_row);
  pp.x_perm = x_perm;
  pp.cap = cap;
  CHECK(hip_status(moe::launch_gather(pp, st), "row gather launch"));
  // routed experts
  FfnBwd r;
  r.x = x_perm;
  r.offsets = C > 0 ? counts : offsets;
  r.groups = s->E_local;
  r.rows = cap;
  r.rows_hint = expected_rows(s);
  r.seg_stride = C;
  r.d = d;
  r.F = F;
  r.w13 = w13;
  r.w2 = w2;
  r.dy = dy_perm;
  r.dx = dx_perm;
  r.dw13 = dw13;
  r.dw2 = dw2;
  r.scratch = scratch;
  CHECK(ffn_backward(r, st));
  // shared expert: one segment of all T token rows, output gradient dout itself
  if (Fs > 0) {
    FfnBwd h;
    h.x = x;
    h.offsets = seg;
    h.groups = 1;
    h.rows = T;
    h.rows_hint = T;
    h.d = d;
    h.F = Fs;
    h.w13 = ws13;
    h.w2 = ws2;
    h.dy = dout;
    h.dx = dx_shared;
    h.dw13 = dws13;
    h.dw2 = dws2;
    h.scratch = scratch;
    CHECK(ffn_backward(h, st));
  }
  // router: dx_router = dlogits w_router (w_router [E][d] read as the transposed operand)
  moe::GemmBwdProblem g{};
  g.mode = moe::BWD_ROWS;
  g.x_mn = false;
  g.w_mn = true;
  g.offsets = seg;
  g.groups = 1;
  g.max_rows = T;
  g.rows_hint = T;
  g.X = dlogits;
  g.ldx = E;
  g.W = static_cast<const moe::bf16_t*>(w_router);
  g.ldw = d;
  g.N = d;
  g.K = E;
  g.Y = dx_router;
  g.ldy = d;
  CHECK(hip_status(moe::launch_gemm_bwd(g, st), "router dx launch"));
  // dw_router = dlogits^T x: float32 partials over token chunks (the K split), summed in
  // chunk order and rounded once
  moe::GemmBwdProblem w = g;
  w.mode = moe::BWD_KSEG;
  w.x_mn = w.w_mn = true;
  w.offsets = at<int32_t>(ws, B.segk);
  w.groups = wr_groups;
  w.X = dlogits;
  w.ldx = E;
  w.W = static_cast<const moe::bf16_t*>(x);
  w.ldw = d;
  w.M = E;
  w.N = d;
  w.Y = nullptr;
  w.Yf = at<float>(ws, B.wr_parts);
  w.ldy = d;
  w.y_group_stride = (int64_t)E * d;
  CHECK(hip_status(moe::launch_gemm_bwd(w, st), "router weight gradient launch"));
  CHECK(hip_status(moe::launch_sum_partials(w.Yf, wr_groups, (int64_t)E * d, static_cast<moe::bf16_t*>(dw_router), st),
                   "router weight gradient sum launch"));
  // dx: the token's expert-row gradients in slot order, then the shared expert's, then the router's
  moe::UnpermuteSumProblem u{};
  u.rows = dx_perm;
  u.slot_row = slot_row;
  u.extra0 = dx_shared;
  u.extra1 = dx_router;
  u.out = static_cast<moe::bf16_t*>(dx);
  u.T = T;
  u.cap = cap;
  u.d = d;
  u.top_k = s->top_k;
  CHECK(hip_status(moe::launch_unpermute_sum(u, st), "row gradient sum launch"));
  return ok();
}

int moe_combine(const moe_shape_t* shape, const void* y_perm, const int32_t* slot_row, const float* topk_w,
                const void* shared_y, void* out, void* stream) {
  CHECK(check_shape(shape));
  if (shape->T == 0) return ok();
  CHECK(check_ptr(y_perm, 16, "y_perm"));
  CHECK(check_ptr(slot_row, 4, "slot_row"));
  CHECK(check_ptr(topk_w, 4, "topk_w"));
  if (shared_y) CHECK(check_ptr(shared_y, 16, "shared_y"));
  CHECK(check_ptr(out, 16, "out"));
  CHECK(do_combine(shape, y_perm, slot_row, topk_w, shared_y, out, as_stream(stream)));
  return ok();
}

int moe_layer_forward_traced(const moe_shape_t* shape, const void* x, const void* w_router, const float* bias,
                             const void* w13, const void* w2, const void* ws13, const void* ws2, void* out,
                             void* ws, size_t ws_bytes, void* const* events, void* stream) {
  CHECK(check_shape(shape));
  if (shape->E_local > moe::kMaxGroups)
    return fail(MOE_ERR_UNSUPPORTED, "E_local (%d) > %d", shape->E_local, moe::kMaxGroups);
  if (bias && shape->gate != MOE_GATE_SOFTMAX)
    return fail(MOE_ERR_UNSUPPORTED, "a router bias is only defined for softmax gating");
  if (shape->T == 0) {
    // nothing to compute; the events are still recorded, back to back (empty intervals)
    if (events)
      for (int i = 0; i <= MOE_STEP_COUNT_; ++i)
        if (events[i])
          CHECK(hip_status(hipEventRecord(static_cast<hipEvent_t>(events[i]), as_stream(stream)), "hipEventRecord"));
    return ok();
  }
  CHECK(check_ptr(x, 16, "x"));
  CHECK(check_ptr(w_router, 16, "w_router"));
  if (bias) CHECK(check_ptr(bias, 4, "bias"));
  CHECK(check_ptr(w13, 16, "w13"));
  CHECK(check_ptr(w2, 16, "w2"));
  if (shape->F_shared > 0) {
    CHECK(check_ptr(ws13, 16, "ws13"));
    CHECK(check_ptr(ws2, 16, "ws2"));
  }
  CHECK(check_ptr(out, 16, "out"));
  if ((shape->fusion & MOE_FUSE_GATHER) && !gather_fits(shape))
    return fail(MOE_ERR_UNSUPPORTED, "MOE_FUSE_GATHER needs T * d * 2 (%lld) < 2^32",
                (long long)(shape->T * (int64_t)shape->d * 2));
  CHECK(check_ws(shape, MOE_WS_LAYER, ws, ws_bytes));

  const LayerLayout L = layer_layout(shape);
  hipStream_t st = as_stream(stream);
  g_events = events;
  g_event_stream = st;
  Marker mark = events ? mark_event : nullptr;
  int32_t* topk_idx = at<int32_t>(ws, L.region[MOE_REGION_TOPK_IDX]);
  float* topk_w = at<float>(ws, L.region[MOE_REGION_TOPK_W]);
  int32_t* counts = at<int32_t>(ws, L.region[MOE_REGION_COUNTS]);
  int32_t* offsets = at<int32_t>(ws, L.region[MOE_REGION_OFFSETS]);
  int32_t* row_token = at<int32_t>(ws, L.region[MOE_REGION_ROW_TOKEN]);
  int32_t* slot_row = at<int32_t>(ws, L.region[MOE_REGION_SLOT_ROW]);
  void* x_perm = at<void>(ws, L.region[MOE_REGION_X_PERM]);
  void* y_perm = at<void>(ws, L.region[MOE_REGION_Y_PERM]);
  void* shared_y = shape->F_shared > 0 ? at<void>(ws, L.region[MOE_REGION_SHARED_Y]) : nullptr;

  if (mark) CHECK(mark(MOE_STEP_ROUTER_GEMM));
  CHECK(do_route(shape, x, w_router, bias, topk_idx, topk_w, nullptr, at<float>(ws, L.logits), st, mark));
  // the permutation folded into the up-projection's copies: its token rows are read from x
  // through row_token (no x_perm round trip), where per-lane 32-bit offsets reach all of x
  const bool fused_gather = fuse_gather(shape);
  // the combine folded into the down-projection: gate-weighted rows added into f32 token rows
  const bool fused_combine = fuse_combine(shape);
  float* acc32 = fused_combine ? at<float>(ws, L.acc32) : nullptr;
  float* row_weight = fused_combine ? at<float>(ws, L.row_weight) : nullptr;
  if (mark) CHECK(mark(MOE_STEP_HISTOGRAM));
  CHECK(do_permute(shape, topk_idx, x, counts, offsets, row_token, slot_row, fused_gather ? nullptr : x_perm,
                   at<void>(ws, L.perm_ws), st, mark, topk_w, row_weight));
  if (fused_combine)
    CHECK(hip_status(moe::launch_zero_f32(acc32, shape->T * (int64_t)shape->d, st), "accumulator clear launch"));
  // a shared expert as wide as the routed ones runs inside the routed launches (its tiles
  // interleaved with the experts'), otherwise in launches of its own
  const bool merged = shape->F_shared > 0 && shape->F_shared == shape->F;
  SharedOperands so;
  if (merged) {
    so.x = x;
    so.w13 = ws13;
    so.w2 = ws2;
    so.act = at<void>(ws, L.act_s);
    so.y = shared_y;
    so.T = shape->T;
  }
  Scatter routed_scatter, shared_scatter;
  if (fused_combine) {
    routed_scatter = Scatter{acc32, row_token, row_weight, shape->T};
    shared_scatter = Scatter{acc32, nullptr, nullptr, shape->T};
  }
  if (mark) CHECK(mark(MOE_STEP_FFN_UP));
  Gather gather;
  if (fused_gather) {
    gather.row_index = row_token;
    gather.x_rows = shape->T;
  }
  const int64_t rows_hint = expected_rows(shape);
  const int C = shape->expert_capacity;
  // the masked-decode layout hands the GEMM the per-expert counts and the segment stride
  CHECK(do_ffn(fused_gather ? x : x_perm, C > 0 ? counts : offsets, shape->E_local, capacity(shape), w13, w2,
               shape->d, shape->F, at<void>(ws, L.act), y_perm, st, mark, MOE_STEP_FFN_DOWN,
               merged ? &so : nullptr, gather, rows_hint, C, routed_scatter));
  if (mark) CHECK(mark(MOE_STEP_SHARED_UP));
  if (shape->F_shared > 0 && !merged)
    CHECK(do_ffn(x, nullptr, 1, shape->T, ws13, ws2, shape->d, shape->F_shared, at<void>(ws, L.act_s), shared_y,
                 st, mark, MOE_STEP_SHARED_DOWN, nullptr, Gather{}, 0, 0, shared_scatter));
  else if (mark)
    CHECK(mark(MOE_STEP_SHARED_DOWN));
  if (mark) CHECK(mark(MOE_STEP_COMBINE));
  if (fused_combine)
    CHECK(hip_status(moe::launch_round_bf16(acc32, static_cast<moe::bf16_t*>(out), shape->T * (int64_t)shape->d, st),
                     "accumulator rounding launch"));
  else
    CHECK(do_combine(shape, y_perm, slot_row, topk_w, shared_y, out, st));
  if (mark) CHECK(mark(MOE_STEP_COUNT_));
  g_events = nullptr;
  return ok();
}

int moe_layer_forward(const moe_shape_t* shape, const void* x, const void* w_router, const float* bias,
                      const void* w13, const void* w2, const void* ws13, const void* ws2, void* out, void* ws,
                      size_t ws_bytes, void* stream) {
  return moe_layer_forward_traced(shape, x, w_router, bias, w13, w2, ws13, ws2, out, ws, ws_bytes, nullptr,
                                  stream);
}

}  // extern "C"
