// Host-only size arithmetic of the kernels' launches and workspaces (no device code): the
// router-logits tile and K split, and the permutation workspace layout.  Kept apart from the
// device sources so the ABI's validation and workspace layer also builds as plain host C++.
#include "kernels.hpp"

namespace moe {

// Router-logits tile: the whole expert row of 256 or more experts in one tile (128 x 256, 8 waves)
// or 128 of them (64 x 128, 4 waves), with K split only as far as needed to reach one workgroup per
// compute unit.  Measured (logits GEMM + gate, token rows read from HBM): DeepSeek-V3 shape
// (8192 x 256 x 7168) 128 x 256 tiles with 4 partials 59.4 us against 69.2 for 256 x 256 tiles with
// 8; skewed shape (16384 x 128 x 2048) 64 x 128 unsplit 37.5 us against 46.6 for 256 x 256 with 4.
// Fewer rows or experts: 64 x 64.
TileShape f32_tile(int64_t rows, int n) {
  if (rows >= 4096 && n >= 256) return {128, 256, 64};
  if (rows >= 4096 && n >= 128) return {64, 128, 64};
  return {64, 64, 64};
}

int logits_splits(int64_t T, int E, int K) {
  constexpr int64_t kTarget = 256;                         // compute units of an MI355X
  constexpr int64_t kMaxSplits = 16;                       // bounds the partials the gate adds
  const TileShape t = f32_tile(T, E);
  const int64_t base = ((T + t.bm - 1) / t.bm) * ((E + t.bn - 1) / t.bn);
  const int64_t nk = (K + t.bk - 1) / t.bk;
  if (base <= 0 || nk <= 1) return 1;
  int64_t s = (kTarget + base - 1) / base;
  s = s < nk ? s : nk;
  s = s < kMaxSplits ? s : kMaxSplits;
  if (s <= 1) return 1;
  const int64_t chunk = (nk + s - 1) / s;
  return (int)((nk + chunk - 1) / chunk);                // every chunk non-empty
}

int64_t permute_supers(int64_t T) {
  constexpr int64_t sc = (int64_t)kPermChunk * kPermSuper;
  return (T + sc - 1) / sc;
}

PermuteWs permute_ws(int64_t T, int E_local) {
  auto al = [](size_t v) { return (v + 255) / 256 * 256; };
  PermuteWs w;
  const size_t table = al((size_t)permute_supers(T) * E_local * sizeof(int32_t));
  const size_t chunks = (size_t)permute_supers(T) * kPermSuper * E_local;
  w.super_count = 0;
  w.super_base = table;
  w.totals = 2 * table;
  w.chunk_mask = w.totals + al((size_t)E_local * sizeof(int32_t));
  w.chunk_base = w.chunk_mask + al(chunks * sizeof(uint64_t));
  w.bytes = w.chunk_base + al(chunks * sizeof(int32_t));
  return w;
}

}  // namespace moe
