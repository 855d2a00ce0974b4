// Host-side checks of the C ABI built with AddressSanitizer and UndefinedBehaviorSanitizer
// (launchers stubbed, see stubs.cpp): the shape / pointer / workspace validation table, the
// T = 0 paths, workspace sizes and region offsets of the five workloads and of shapes at the
// stated limits, and valid calls that run the whole host-side setup up to their first launch.
// Prints one line per failed check and "ALL OK" when none failed.
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "../../include/moe.h"

extern int g_launches, g_events;

static int g_fail = 0;
#define EXPECT(cond, ...)                         \
  do {                                            \
    if (!(cond)) {                                \
      ++g_fail;                                   \
      printf("FAIL line %d: ", __LINE__);         \
      printf(__VA_ARGS__);                        \
      printf(" [%s]\n", moe_last_error());        \
    }                                             \
  } while (0)

static void* const FAKE = reinterpret_cast<void*>(0x100000);
static void* const MIS = reinterpret_cast<void*>(0x100002);

static moe_shape_t base() {
  moe_shape_t s;
  memset(&s, 0, sizeof s);
  s.T = 64; s.d = 64; s.E = 8; s.top_k = 2; s.e_begin = 0; s.E_local = 8; s.F = 64; s.F_shared = 0;
  s.gate = MOE_GATE_SOFTMAX; s.n_group = 1; s.topk_group = 1; s.renormalize = 1; s.routed_scale = 1.0f;
  return s;
}

static int layer(const moe_shape_t* s, void* x = FAKE, void* ws = FAKE, size_t ws_bytes = 0, const float* bias = nullptr,
                 void* out = FAKE, void* ws13 = nullptr) {
  return moe_layer_forward(s, x, FAKE, bias, FAKE, FAKE, ws13, ws13, out, ws, ws_bytes, nullptr);
}

static void shape_case(moe_shape_t s, int status, const char* needle) {
  const int st = layer(&s);
  EXPECT(st == status && strstr(moe_last_error(), needle), "shape case '%s': status %d", needle, st);
  EXPECT(moe_workspace_size(&s, MOE_WS_LAYER) == 0, "workspace size of an invalid shape '%s'", needle);
}

int main() {
  moe_shape_t s;
  // ---- shape validation ----
  s = base(); s.d = 60; shape_case(s, MOE_ERR_UNSUPPORTED, "d (60) % 8 != 0");
  s = base(); s.F = 12; shape_case(s, MOE_ERR_UNSUPPORTED, "F (12) % 8 != 0");
  s = base(); s.F_shared = -8; shape_case(s, MOE_ERR_INVALID_ARG, "F_shared (-8) < 0");
  s = base(); s.E = 2000; shape_case(s, MOE_ERR_UNSUPPORTED, "E (2000) outside [1, 1024]");
  s = base(); s.top_k = 9; shape_case(s, MOE_ERR_UNSUPPORTED, "top_k (9)");
  s = base(); s.E = 64; s.top_k = 17; shape_case(s, MOE_ERR_UNSUPPORTED, "top_k (17)");
  s = base(); s.e_begin = 4; s.E_local = 5; shape_case(s, MOE_ERR_INVALID_ARG, "local slice");
  s = base(); s.E_local = 0; shape_case(s, MOE_ERR_INVALID_ARG, "local slice");
  s = base(); s.e_begin = 2147483000; shape_case(s, MOE_ERR_INVALID_ARG, "local slice");
  s = base(); s.n_group = 3; shape_case(s, MOE_ERR_INVALID_ARG, "E (8) % n_group (3) != 0");
  s = base(); s.n_group = 8; s.topk_group = 4; shape_case(s, MOE_ERR_INVALID_ARG, "group size");
  s = base(); s.n_group = 4; s.topk_group = 5; shape_case(s, MOE_ERR_INVALID_ARG, "topk_group (5)");
  s = base(); s.E = 16; s.top_k = 6; s.E_local = 16; s.n_group = 4; s.topk_group = 1;
  shape_case(s, MOE_ERR_INVALID_ARG, "< top_k (6)");
  s = base(); s.gate = 7; shape_case(s, MOE_ERR_UNSUPPORTED, "gate (7)");
  s = base(); s.renormalize = 2; shape_case(s, MOE_ERR_INVALID_ARG, "renormalize (2)");
  s = base(); s.routed_scale = __builtin_nanf(""); shape_case(s, MOE_ERR_INVALID_ARG, "routed_scale");
  s = base(); s.T = -1; shape_case(s, MOE_ERR_INVALID_ARG, "T (-1) < 0");
  s = base(); s.T = (int64_t)1 << 30; shape_case(s, MOE_ERR_UNSUPPORTED, "T * top_k");
  s = base(); s.T = INT64_MAX / 2; shape_case(s, MOE_ERR_UNSUPPORTED, "T * top_k");
  s = base(); s.expert_capacity = -1; shape_case(s, MOE_ERR_INVALID_ARG, "expert_capacity (-1) < 0");
  s = base(); s.expert_capacity = 1 << 28; shape_case(s, MOE_ERR_UNSUPPORTED, "E_local * expert_capacity");
  s = base(); s.fusion = MOE_FUSE_COMBINE; shape_case(s, MOE_ERR_INVALID_ARG, "fusion (0x2)");
  s = base(); s.fusion = MOE_FUSION_SET | 0x4; shape_case(s, MOE_ERR_INVALID_ARG, "fusion (0x14)");
  EXPECT(layer(nullptr) == MOE_ERR_INVALID_ARG && strstr(moe_last_error(), "shape is NULL"), "null shape");

  // ---- pointers and workspace ----
  s = base();
  const size_t need = moe_workspace_size(&s, MOE_WS_LAYER);
  EXPECT(need > 0 && need % 256 == 0, "layer workspace %zu", need);
  EXPECT(layer(&s, nullptr) == MOE_ERR_INVALID_ARG && strstr(moe_last_error(), "x is NULL"), "x NULL");
  EXPECT(moe_layer_forward(&s, FAKE, FAKE, nullptr, MIS, FAKE, nullptr, nullptr, FAKE, FAKE, need, nullptr) ==
             MOE_ERR_INVALID_ARG && strstr(moe_last_error(), "16-byte aligned"), "w13 misaligned");
  EXPECT(layer(&s, FAKE, nullptr, need) == MOE_ERR_WORKSPACE, "workspace NULL");
  EXPECT(layer(&s, FAKE, FAKE, need - 1) == MOE_ERR_WORKSPACE, "workspace too small");
  EXPECT(layer(&s, FAKE, MIS, need) == MOE_ERR_INVALID_ARG, "workspace misaligned");
  moe_shape_t sh = base(); sh.F_shared = 64;
  EXPECT(layer(&sh, FAKE, FAKE, (size_t)1 << 40) == MOE_ERR_INVALID_ARG && strstr(moe_last_error(), "ws13 is NULL"),
         "ws13 NULL");
  moe_shape_t sg = base(); sg.gate = MOE_GATE_SIGMOID;
  EXPECT(layer(&sg, FAKE, FAKE, need, static_cast<const float*>(FAKE)) == MOE_ERR_UNSUPPORTED, "sigmoid bias");

  // ---- components ----
  EXPECT(moe_route(&s, FAKE, FAKE, nullptr, nullptr, static_cast<float*>(FAKE), nullptr, FAKE, (size_t)1 << 40,
                   nullptr) == MOE_ERR_INVALID_ARG, "route topk_idx NULL");
  EXPECT(moe_route(&s, FAKE, FAKE, nullptr, static_cast<int32_t*>(FAKE), static_cast<float*>(FAKE), nullptr, FAKE,
                   16, nullptr) == MOE_ERR_WORKSPACE, "route workspace");
  int32_t* I = static_cast<int32_t*>(FAKE);
  EXPECT(moe_permute(&s, I, FAKE, I, I, I, static_cast<int32_t*>(MIS), FAKE, FAKE, (size_t)1 << 40, nullptr) ==
             MOE_ERR_INVALID_ARG, "permute slot_row misaligned");
  EXPECT(moe_permute_noalloc(&s, nullptr, FAKE, I, I, I, I, FAKE, nullptr) == MOE_ERR_INVALID_ARG,
         "noalloc topk_idx NULL");
  moe_shape_t big = base(); big.T = 1 << 16; big.E = 128; big.E_local = 128; big.top_k = 8;
  EXPECT(moe_permute_noalloc(&big, I, FAKE, I, I, I, I, FAKE, nullptr) == MOE_ERR_UNSUPPORTED, "noalloc size");
  EXPECT(moe_grouped_ffn(&s, FAKE, nullptr, FAKE, FAKE, FAKE, FAKE, (size_t)1 << 40, nullptr) == MOE_ERR_INVALID_ARG,
         "ffn offsets NULL");
  EXPECT(moe_combine(&s, FAKE, I, static_cast<float*>(FAKE), MIS, FAKE, nullptr) == MOE_ERR_INVALID_ARG,
         "combine shared_y misaligned");

  // ---- T = 0: no-ops (the traced form records its events back to back) ----
  moe_shape_t z = base(); z.T = 0;
  EXPECT(moe_layer_forward(&z, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0,
                           nullptr) == MOE_OK, "T = 0 layer");
  void* ev[MOE_STEP_COUNT_ + 1];
  for (int i = 0; i <= MOE_STEP_COUNT_; ++i) ev[i] = FAKE;
  const int e0 = g_events;
  EXPECT(moe_layer_forward_traced(&z, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                  0, ev, nullptr) == MOE_OK && g_events - e0 == MOE_STEP_COUNT_ + 1,
         "T = 0 traced records %d events", g_events - e0);
  ev[3] = nullptr;                                         // a NULL entry is skipped
  const int e1 = g_events;
  EXPECT(moe_layer_forward_traced(&z, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                  0, ev, nullptr) == MOE_OK && g_events - e1 == MOE_STEP_COUNT_,
         "T = 0 traced with a NULL entry records %d events", g_events - e1);
  EXPECT(moe_permute_noalloc(&z, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr) == MOE_OK,
         "T = 0 noalloc");

  // ---- workspace sizes and region offsets: the five workloads and shapes at the limits ----
  moe_shape_t wl[7];
  for (int i = 0; i < 7; ++i) wl[i] = base();
  wl[0].T = 256; wl[0].d = 512; wl[0].E = 8; wl[0].top_k = 2; wl[0].F = 1024; wl[0].E_local = 8;
  wl[1].T = 4096; wl[1].d = 4096; wl[1].E = 8; wl[1].top_k = 2; wl[1].F = 14336; wl[1].E_local = 8;
  wl[2].T = 8192; wl[2].d = 7168; wl[2].E = 256; wl[2].top_k = 8; wl[2].F = 2048; wl[2].E_local = 32;
  wl[2].F_shared = 2048; wl[2].gate = MOE_GATE_SIGMOID; wl[2].n_group = 8; wl[2].topk_group = 4;
  wl[2].routed_scale = 2.5f;
  wl[3].T = 16384; wl[3].d = 2048; wl[3].E = 128; wl[3].top_k = 8; wl[3].F = 768; wl[3].E_local = 128;
  wl[4].T = 64; wl[4].d = 7168; wl[4].E = 384; wl[4].top_k = 8; wl[4].F = 2048; wl[4].E_local = 48;
  wl[4].F_shared = 2048; wl[4].gate = MOE_GATE_SIGMOID;
  wl[5].T = ((int64_t)1 << 31) / 16 - 1; wl[5].d = 8; wl[5].E = 1024; wl[5].top_k = 16; wl[5].E_local = 1024;
  wl[5].F = 8;                                                     // T * top_k just below 2^31
  wl[6] = wl[4]; wl[6].expert_capacity = 8; wl[6].fusion = MOE_FUSION_SET | MOE_FUSE_GATHER | MOE_FUSE_COMBINE;
  for (int i = 0; i < 7; ++i) {
    size_t prev = 0;
    for (int k = MOE_WS_ROUTE; k <= MOE_WS_LAYER_BWD; ++k) {
      const size_t n = moe_workspace_size(&wl[i], k);
      EXPECT(n > 0 && n % 256 == 0, "workload %d kind %d size %zu", i, k, n);
    }
    const size_t total = moe_workspace_size(&wl[i], MOE_WS_LAYER);
    for (int r = 0; r < MOE_REGION_COUNT_; ++r) {
      const size_t off = moe_workspace_offset(&wl[i], r);
      EXPECT(off != (size_t)-1 && off % 256 == 0 && off >= prev && off <= total, "workload %d region %d", i, r);
      prev = off;
    }
  }
  EXPECT(moe_workspace_offset(&wl[2], MOE_REGION_COUNT_) == (size_t)-1, "region out of range");
  EXPECT(moe_workspace_size(&wl[2], 99) == 0, "kind out of range");

  // ---- valid calls: the whole host-side setup, up to the first (stubbed) launch ----
  for (int i = 0; i < 5; ++i) {
    const int l0 = g_launches;
    const size_t n = moe_workspace_size(&wl[i], MOE_WS_LAYER);
    const int st = moe_layer_forward(&wl[i], FAKE, FAKE, nullptr, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, n, nullptr);
    EXPECT(st == MOE_ERR_HIP && g_launches == l0 + 1 && strstr(moe_last_error(), "stub launch"),
           "workload %d layer reaches its first launch (status %d)", i, st);
    const size_t nb = moe_workspace_size(&wl[i], MOE_WS_LAYER_BWD);
    const int sb = moe_layer_backward(&wl[i], FAKE, FAKE, nullptr, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, n, FAKE, FAKE,
                                      FAKE, FAKE, FAKE, FAKE, FAKE, nb, nullptr);
    EXPECT(sb == MOE_ERR_HIP, "workload %d backward reaches its first launch (status %d)", i, sb);
  }
  EXPECT(moe_permute_noalloc(&s, I, FAKE, I, I, I, I, FAKE, nullptr) == MOE_ERR_HIP, "noalloc scratch lookup");
  {
    // traced, only some events asked for: the first step's event is recorded, then its launch fails
    void* sparse[MOE_STEP_COUNT_ + 1] = {};
    sparse[0] = FAKE;
    sparse[MOE_STEP_FFN_UP] = FAKE;
    const size_t n = moe_workspace_size(&wl[2], MOE_WS_LAYER);
    const int e2 = g_events;
    const int st = moe_layer_forward_traced(&wl[2], FAKE, FAKE, nullptr, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, n,
                                            sparse, nullptr);
    EXPECT(st == MOE_ERR_HIP && g_events - e2 == 1, "sparse traced call (status %d, %d events)", st, g_events - e2);
  }

  if (g_fail == 0) printf("ALL OK\n");
  return g_fail == 0 ? 0 : 1;
}
