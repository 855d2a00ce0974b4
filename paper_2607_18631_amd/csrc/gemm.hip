// Grouped GEMM on gfx950 bf16 MFMA (v_mfma_f32_32x32x16_bf16), fp32 accumulation.
//
//   Y[r, n] = sum_k X[r, k] * W_g[n, k]     for every group g, every row r in [offs[g], offs[g+1])
//
// One launch serves every group (local expert) of a batch: the row segment of group g
// is [offsets[g], offsets[g+1]) -- the monotone [E+1] row-offset array of the paper's
// kernel-generation section -- read from device memory, so the row counts never travel
// to the host.  Each workgroup builds the launch's tile table in LDS (ceil(m_g / BM) x
// n-tiles per group, one block-wide prefix sum), decodes the tiles it will run into a short
// list (one thread per tile), and then walks them persistently.
// Tiles of one group are ordered m-fastest, so the m-tiles sharing a weight tile are
// adjacent, and adjacent tiles go to workgroups of the same XCD (workgroup i runs on XCD
// i mod 8): a weight tile is fetched from HBM once per XCD L2, not once per m-tile.
//
// Data movement: K is consumed in BK-wide slices through a STAGES-deep LDS ring.  Slices
// are copied global -> LDS by the direct-to-LDS loads of gfx950 (global_load_lds_dwordx4:
// lane i of a wave instruction writes bytes [16 i, 16 i + 16) after the wave's LDS base),
// issued STAGES-1 slices ahead, so HBM/L2 latency hides behind the MFMAs of the slices in
// between and no VGPR staging is needed; a slice's copies go out one per MFMA of the K-step
// that follows the barrier that frees their ring slot.  A slice is consumed after `s_waitcnt vmcnt`
// (this wave's copies of it have landed) and a workgroup barrier (everyone's have).
// The barrier also orders the reuse of a ring slot: the slot refilled in iteration kt was
// last read in iteration kt-1, which every wave has finished once it passes the barrier.
//
// LDS layout of a slice: [rows][BK] bf16, row r's 16-byte chunk c stored at chunk
// c ^ f(r), f(r) = (r / (16 / CPR)) % CPR with CPR = BK / 8 chunks per row.  The 16 lanes of
// one ds_read_b128 phase read one logical chunk of 16 consecutive rows and hit 16
// distinct 16-byte bank groups.  The swizzle is applied on the global side: a lane
// fetches the logical chunk that belongs at its fixed LDS position.
//
// Operand roles: the weight tile is the MFMA A operand (rows = output features) and the
// token tile the B operand (columns = tokens), so each lane ends with 4 consecutive
// output features of one token: 8-byte bf16 stores along the output row.
//
// Edges: token rows past the group's end and weight rows past N are clamped to the last
// valid row (their results are never stored); a K tail (K % BK != 0) is fetched from
// clamped addresses and its chunks past K are zeroed in LDS before use.  The 32-row token
// blocks of a tile alternate over the waves, and a wave runs no MFMA for its blocks past
// the group's end, so the ragged last m-tile of an expert costs MFMA time in proportion to
// its live rows (the per-expert row counts of a routed batch scatter around the mean,
// which leaves most experts with one mostly empty m-tile).
//
// Variants of the same body: equal-stride row segments [g * seg_stride, + count_g) (the
// masked-decode form of the same section: capacity offsets plus valid counts); gathered
// token rows (the permute folded into the prologue: row r of the tile is X row
// row_index[r]); and the scatter epilogue (the weighted combine folded into the epilogue:
// rows added, times their gate, into float32 token rows with atomics).
#include <algorithm>
#include <cmath>
#include <type_traits>

#include "common.hpp"
#include "gemm_device.hpp"
#include "kernels.hpp"

namespace moe {

// device properties, queried once per device (std::call_once on the first launch there)
struct DevInfo {
  std::once_flag once;
  int cus = 256;
  int lds = 65536;
};
static DevInfo g_dev[kMaxDevices];

static const DevInfo* dev_info() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  DevInfo& d = g_dev[dev];
  std::call_once(d.once, [&] {
    int n = 0, l = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0) d.cus = n;
    if (hipDeviceGetAttribute(&l, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) == hipSuccess && l > 0) d.lds = l;
  });
  return &d;
}
int cu_count() {
  const DevInfo* d = dev_info();
  return d ? d->cus : 256;
}
int lds_limit() {
  const DevInfo* d = dev_info();
  return d ? d->lds : 65536;
}

int kernel_occupancy(OccCache& c, const void* fn, int nth, size_t lds, hipError_t& err) {
  err = hipSuccess;
  int dev = 0;
  if ((err = hipGetDevice(&dev)) != hipSuccess) return 0;
  if (dev < 0 || dev >= kMaxDevices) {
    err = hipErrorInvalidDevice;
    return 0;
  }
  std::call_once(c.once[dev], [&] {
    int occ = 0;
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e == hipSuccess) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, fn, nth, lds);
    c.err[dev] = e;
    c.per_cu[dev] = occ > 0 ? occ : 1;
  });
  err = c.err[dev];
  return err == hipSuccess ? c.per_cu[dev] : 0;
}

namespace {

// epilogues whose weight tile pairs gate rows [0, N) with up rows [N, 2N)
constexpr bool swiglu_pairs(int epi) { return epi == EPI_SWIGLU || epi == EPI_SWIGLU_BWD; }

#ifndef MOE_BAND_M
#define MOE_BAND_M 8
#endif
constexpr int BAND_M = MOE_BAND_M;   // m-tiles per band of the tile order





// ---------------------------------------------------------------------------------------
// Tile table, tile decoding, slice copies, epilogue
// ---------------------------------------------------------------------------------------

// Tiles of one launch: `groups` row segments of BM-row tiles x tiles_n output tiles each,
// plus tiles_x tiles of the optional extra group, `total` in all.  s_off / s_tp live in LDS.
// With a K split (ksplit > 1, one group, no extra group) the tile space is ksplit copies of
// the (m, n) tiles, chunk c covering K slices [c * kchunk, min(nk, (c + 1) * kchunk)); chunk is
// the slowest index, so the workgroups of one XCD work on one K chunk of the weights.
struct TileSpace {
  int groups, tiles_n, tiles_x, total;
  int bmx;                   // m-tile height of the extra group
  int base_total;            // (m, n) tiles
  int nk, kchunk;            // K slices; slices per chunk
  int seg_stride;            // > 0: group g owns rows [g * seg_stride, g * seg_stride + s_off[g])
  const int* s_off;          // [groups + 1] row offsets clamped to [0, max_rows] (or valid lengths)
  const int* s_tp;           // [groups + 1] first tile of each group; s_tp[groups] = grouped tiles
  __device__ int seg_begin(int g) const { return seg_stride > 0 ? g * seg_stride : s_off[g]; }
  __device__ int seg_end(int g) const { return seg_stride > 0 ? g * seg_stride + s_off[g] : s_off[g + 1]; }
};

// Build the launch's tile table in LDS (every thread of the block calls this).
template <int NTH, int BM, int BK>
__device__ TileSpace build_tile_space(const GemmProblem& p, int outn, int* s_off, int* s_tp, int* s_tmp) {
  const int tid = threadIdx.x;
  TileSpace ts;
  ts.tiles_n = (p.N + outn - 1) / outn;
  int groups = p.groups;
  ts.seg_stride = 0;
  if (p.offsets && p.seg_stride > 0) {
    // equal-stride segments: the valid length of each, clamped to [0, seg_stride] (the
    // launcher keeps groups * seg_stride <= max_rows)
    ts.seg_stride = p.seg_stride;
    for (int g = tid; g < groups; g += NTH) s_off[g] = min(max(p.offsets[g], 0), p.seg_stride);
  } else if (p.offsets) {
    // clamp to [0, max_rows]: any offsets content keeps every access inside the buffers
    const int cap = (int)p.max_rows;
    for (int g = tid; g <= groups; g += NTH) s_off[g] = min(max(p.offsets[g], 0), cap);
  } else {
    groups = 1;
    if (tid == 0) { s_off[0] = 0; s_off[1] = (int)p.rows_single; }
  }
  __syncthreads();
  constexpr int PER = (kMaxGroups + NTH - 1) / NTH;
  int loc[PER];
  int lsum = 0;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    int g = tid * PER + i;
    int m = g >= groups ? 0 : ts.seg_stride > 0 ? s_off[g] : max(s_off[g + 1] - s_off[g], 0);
    loc[i] = ((m + BM - 1) / BM) * ts.tiles_n;
    lsum += loc[i];
  }
  int excl;
  const int total_r = block_exclusive_scan<NTH>(lsum, s_tmp, excl);
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    int g = tid * PER + i;
    if (g < groups) s_tp[g] = excl;
    excl += loc[i];
  }
  if (tid == 0) s_tp[groups] = total_r;
  __syncthreads();
  // the extra group's tiles sit among the grouped ones (see extra_position)
  ts.bmx = (p.rows2_tile > 0 && p.rows2_tile < BM) ? p.rows2_tile : BM;
  ts.tiles_x = p.rows2 > 0 ? ((p.rows2 + ts.bmx - 1) / ts.bmx) * ts.tiles_n : 0;
  ts.base_total = total_r + ts.tiles_x;
  ts.nk = (p.K + BK - 1) / BK;
  const int ksplit = p.ksplit > 1 ? p.ksplit : 1;
  ts.kchunk = (ts.nk + ksplit - 1) / ksplit;
  ts.total = ts.base_total * ksplit;
  ts.groups = groups;
  ts.s_off = s_off;
  ts.s_tp = s_tp;
  return ts;
}


// One tile: token rows [row0, min(row0 + BM, row_end)) of operand X against output tile ni
// of the weights W, results into Y.
struct TileDesc {
  int row0, row_end, ni;
  int kb, ke, kc;            // K slices [kb, ke) of K chunk kc
  const int32_t* rows;       // gathered rows: tile row r is X row rows[row0 + r] (else row0 + r)
  const int32_t* stok;       // EPI_SCATTER: token of each row (nullptr: the row itself)
  const float* sw;           // EPI_SCATTER: weight of each row (nullptr: 1)
  const bf16_t* X;
  const bf16_t* W;
  void* Y;
};

#ifndef MOE_EXTRA_BLOCKS
#define MOE_EXTRA_BLOCKS 1
#endif
// Where the extra group's (shared expert's) tiles sit among the grouped ones: x_before = extra
// tiles before position t, extra = position t is one.  Workgroup i runs on XCD i % 8 and an XCD
// takes G / 8 consecutive positions per round of the persistent grid, so the extra tiles are
// spread over whole such blocks: every block is all-extra or all-grouped (the last extra block
// may be part-filled, its other positions grouped), which keeps the tiles an XCD runs together
// on shared token and weight panels, while HBM-bound expert blocks and compute-bound shared
// blocks still run side by side on the chip.  Problems with fewer full blocks than extra blocks
// (or grids that are not whole rounds of the 8 XCDs) spread tile by tile.
__device__ __forceinline__ void extra_position(const TileSpace& ts, int t, int& x_before, bool& extra) {
  const int S = ts.tiles_x, T = ts.base_total;
  const int G = gridDim.x;
  const int BS = (MOE_EXTRA_BLOCKS && G % 8 == 0) ? G / 8 : 1;
  const int nbf = T / BS;                                 // full blocks
  const int sb = (S + BS - 1) / BS;                       // blocks the extra tiles fill
  if (S == 0 || BS == 1 || sb > nbf) {
    x_before = (int)((int64_t)t * S / T);
    extra = (int)((int64_t)(t + 1) * S / T) > x_before;
    return;
  }
  const int b = t / BS, o = t - b * BS;
  // extra blocks among the full ones: block b is one iff floor((b+1) sb / nbf) > floor(b sb / nbf)
  const int before = (int)((int64_t)min(b, nbf) * sb / nbf);
  const bool xblock = b < nbf && (int)((int64_t)(b + 1) * sb / nbf) > before;
  const int first = before * BS;                          // extra tiles in earlier blocks
  extra = xblock && first + o < S;
  x_before = min(S, first + (xblock ? o : 0));
}

// A tile's coordinates: rows [row0, row_end) of group g (-1: the extra group), output tile ni,
// K slices [kb, ke) of K chunk kc.  Computed by any thread on its own (no wave-uniform input).
struct TileCode {
  int row0, row_end, ni, kb, ke, kc, g;
};

template <int BM>
__device__ __forceinline__ TileCode tile_code(const GemmProblem& p, const TileSpace& ts, int tile) {
  TileCode c;
  c.kc = tile / ts.base_total;
  tile -= c.kc * ts.base_total;
  c.kb = c.kc * ts.kchunk;
  c.ke = min(ts.nk, c.kb + ts.kchunk);
  int x_before;
  bool extra;
  extra_position(ts, tile, x_before, extra);
  int row0g, local;
  if (extra) {
    row0g = 0;
    c.row_end = p.rows2;
    local = x_before;
    c.g = -1;
  } else {
    const int t = tile - x_before;                        // index among the grouped tiles
    int lo = 0, hi = ts.groups;                           // s_tp[groups] == grouped tiles > t
    while (hi - lo > 1) {
      int mid = (lo + hi) >> 1;
      if (ts.s_tp[mid] <= t) lo = mid; else hi = mid;
    }
    c.g = lo;
    row0g = ts.seg_begin(lo);
    c.row_end = ts.seg_end(lo);
    local = t - ts.s_tp[lo];
  }
  const int bmg = extra ? ts.bmx : BM;                  // m-tile height of this group
  const int mt = (c.row_end - row0g + bmg - 1) / bmg;
  // banded order: bands of up to BAND_M m-tiles; inside a band m-fastest, then n.  The
  // 32 adjacent tiles one XCD runs at a time then share BAND_M token panels and
  // 32 / BAND_M weight panels (groups with few m-tiles reduce to plain m-fastest order)
  const int band = local / (BAND_M * ts.tiles_n);
  const int bm0 = band * BAND_M;
  const int bmt = min(BAND_M, mt - bm0);
  const int in_band = local - band * BAND_M * ts.tiles_n;
  const int mi = bm0 + in_band % bmt;
  c.ni = in_band / bmt;
  c.row0 = row0g + mi * bmg;
  if (bmg < BM) c.row_end = min(c.row0 + bmg, c.row_end);   // the extra group's shorter tiles
  return c;
}

// The tile of a wave-uniform code (values moved to scalar registers) with its operand pointers.
__device__ __forceinline__ TileDesc tile_desc(const GemmProblem& p, TileCode c) {
  TileDesc d;
  d.row0 = __builtin_amdgcn_readfirstlane(c.row0);
  d.row_end = __builtin_amdgcn_readfirstlane(c.row_end);
  d.ni = __builtin_amdgcn_readfirstlane(c.ni);
  d.kb = __builtin_amdgcn_readfirstlane(c.kb);
  d.ke = __builtin_amdgcn_readfirstlane(c.ke);
  d.kc = __builtin_amdgcn_readfirstlane(c.kc);
  const int g = __builtin_amdgcn_readfirstlane(c.g);
  if (g < 0) {
    d.W = p.W2;
    d.X = p.X2;
    d.Y = p.Y2;
    d.rows = nullptr;
    d.stok = nullptr;
    d.sw = nullptr;
  } else {
    d.W = p.W + (int64_t)g * p.w_group_stride;
    d.X = p.X;
    d.Y = p.Y;
    d.rows = p.row_index;
    d.stok = p.scatter_token;
    d.sw = p.scatter_weight;
  }
  return d;
}

// Tiles a workgroup decodes once at its start (one thread per tile) and keeps in LDS; the
// position of its round r is r G + slot in even rounds, r G + G - 1 - slot in odd ones.
constexpr int kTileList = 64;
__device__ __forceinline__ int round_position(int r, int slot) {
  const int G = gridDim.x;
  return r * G + ((r & 1) ? G - 1 - slot : slot);
}

// Copies of one K slice of a tile into a ring slot, spread over NW waves.  Per tile, a
// wave-uniform base (scalar registers) per copy instruction and a fixed per-lane 32-bit byte
// offset (row * ld + logical chunk), so a full slice's copies cost one scalar add each and
// no vector ALU.  The W instruction j is uniformly in the gate or the up half of a SwiGLU
// tile.  Token rows past the tile's end and weight rows past N are clamped to the last valid
// row.
template <int BM, int BN, int BK, int NW, int EPI>
struct CopyPlan {
  using Z = Swz<BK>;
  static constexpr int RPI = 1024 / (BK * 2);              // rows one wave instruction fills
  static constexpr int LX = BM / RPI / NW, LW = BN / RPI / NW;
  static constexpr int L = LX + LW;                        // vector-memory ops per wave per slice
  static_assert(LX >= 1 && LW >= 1 && (BM / RPI) % NW == 0 && (BN / RPI) % NW == 0, "tile too small");

  const char* xbase;
  const char* wsb[LW];
  uint32_t xoff[LX], woff[LW];
  int xchunk[LX], wchunk[LW];

  __device__ __forceinline__ void setup(const GemmProblem& p, const TileDesc& t, int wave, int lane) {
    const int li_row = lane / Z::CPR, li_pc = lane % Z::CPR;
    const int K = p.K;
    const int last = t.row_end - 1 - t.row0;
    if (t.rows) {
      // gathered rows: the lane's own source row (the launcher keeps x_rows * ldx * 2 < 2^32)
      xbase = reinterpret_cast<const char*>(t.X);
      const int top = (int)p.x_rows - 1;
#pragma unroll
      for (int j = 0; j < LX; ++j) {
        const int r = (wave + NW * j) * RPI + li_row;
        xchunk[j] = li_pc ^ Z::f(r);
        const int src = min(max(t.rows[t.row0 + min(r, last)], 0), top);
        xoff[j] = (uint32_t)((int64_t)src * p.ldx * 2 + xchunk[j] * 16);
      }
    } else {
      xbase = reinterpret_cast<const char*>(t.X + (int64_t)t.row0 * p.ldx);
#pragma unroll
      for (int j = 0; j < LX; ++j) {
        const int r = (wave + NW * j) * RPI + li_row;         // tile row
        xchunk[j] = li_pc ^ Z::f(r);
        xoff[j] = (uint32_t)(min(r, last) * p.ldx * 2 + xchunk[j] * 16);
      }
    }
#pragma unroll
    for (int j = 0; j < LW; ++j) {
      const int r = (wave + NW * j) * RPI + li_row;
      wchunk[j] = li_pc ^ Z::f(r);
      if (swiglu_pairs(EPI)) {
        const int half = ((wave + NW * j) * RPI) >= BN / 2;  // uniform per instruction
        const int f0 = t.ni * (BN / 2);
        const int f = min(f0 + (r - half * (BN / 2)), p.N - 1);
        wsb[j] = reinterpret_cast<const char*>(t.W + ((int64_t)f0 + half * p.N) * K);
        woff[j] = (uint32_t)((f - f0) * K * 2 + wchunk[j] * 16);
      } else {
        const int f0 = t.ni * BN;
        const int f = min(f0 + r, p.N - 1);
        wsb[j] = reinterpret_cast<const char*>(t.W + (int64_t)f0 * K);
        woff[j] = (uint32_t)((f - f0) * K * 2 + wchunk[j] * 16);
      }
    }
  }

  // copy K slice kt into the ring slot at dst (L vector-memory ops of this wave)
  __device__ __forceinline__ void issue(bf16_t* dst, int kt, int wave) const {
    const int k0b = kt * BK * 2;                           // byte offset of the slice
#pragma unroll
    for (int j = 0; j < LX; ++j)
      dma16(reinterpret_cast<const bf16_t*>(xbase + k0b + xoff[j]), dst + (wave + NW * j) * 512);
#pragma unroll
    for (int j = 0; j < LW; ++j)
      dma16(reinterpret_cast<const bf16_t*>(wsb[j] + k0b + woff[j]), dst + BM * BK + (wave + NW * j) * 512);
  }

  // Copy J of K slice kt into the ring slot at dst through a scalar base (the instruction's
  // uniform row block plus the slice's byte offset) and the lane's 32-bit offset: no 64-bit
  // per-lane address arithmetic and no per-lane 64-bit bases held across the K loop.  The
  // compiler does not see these copies; the K loop orders them with its own vmcnt waits and
  // barriers.
  template <int J>
  __device__ __forceinline__ void issue_one_sv(bf16_t* dst, int kt, int wave) const {
    const int k0b = kt * BK * 2;
    if constexpr (J < LX) {
      dma16_sv(xbase + k0b, xoff[J], dst + (wave + NW * J) * 512);
    } else {
      constexpr int JW = J - LX;
      dma16_sv(wsb[JW] + k0b, woff[JW], dst + BM * BK + (wave + NW * JW) * 512);
    }
  }
  template <int J = 0>
  __device__ __forceinline__ void issue_sv(bf16_t* dst, int kt, int wave) const {
    if constexpr (J < L) {
      issue_one_sv<J>(dst, kt, wave);
      issue_sv<J + 1>(dst, kt, wave);
    }
  }

  // the partial last slice (K % BK != 0): chunks past K are fetched from K-8 and zeroed later
  __device__ __forceinline__ void issue_tail(bf16_t* dst, int kt, int wave, int K) const {
    const int k0 = kt * BK;
#pragma unroll
    for (int j = 0; j < LX; ++j) {
      const int back = max(k0 + xchunk[j] * 8 - (K - 8), 0) * 2;
      dma16(reinterpret_cast<const bf16_t*>(xbase + k0 * 2 + xoff[j] - back), dst + (wave + NW * j) * 512);
    }
#pragma unroll
    for (int j = 0; j < LW; ++j) {
      const int back = max(k0 + wchunk[j] * 8 - (K - 8), 0) * 2;
      dma16(reinterpret_cast<const bf16_t*>(wsb[j] + k0 * 2 + woff[j] - back), dst + BM * BK + (wave + NW * j) * 512);
    }
  }
};

// First W-tile row of fragment b of a wave whose sub-tile is column block wn of WGN (each
// wave owns the gate rows and the matching up rows of its features in a SwiGLU tile).
template <int EPI, int BN, int WGN, int FN>
__device__ __forceinline__ int frag_wrow(int wn, int b) {
  if (swiglu_pairs(EPI)) {
    constexpr int HALF_W = BN / 2 / WGN;
    return (b < FN / 2) ? wn * HALF_W + b * 32 : BN / 2 + wn * HALF_W + (b - FN / 2) * 32;
  }
  return wn * (BN / WGN) + b * 32;
}

// silu(g) = g / (1 + e^-g) is taken as g * rcp(1 + e^-g) (v_rcp_f32, 1 ulp) in every epilogue: the
// result is rounded to bf16 next, and an IEEE division costs ~10 VALU instructions per element.
// Store one wave's FM x FN accumulator fragments of tile t.  Lane holds token row
// trow + astride a + (lane & 31) and output features fcol + 32 b + 8 q + 4 (lane >> 5) + 0..3.
// SwiGLU pairs fragment b (gate) with b + FN/2 (up): Y = bf16(silu(gate) * up).
template <int EPI, int FM, int FN>
__device__ __forceinline__ void store_tile(const GemmProblem& p, const f32x16 (&acc)[FM][FN], const TileDesc& t,
                                           int trow, int astride, int fcol, int lane) {
#pragma unroll
  for (int a = 0; a < FM; ++a) {
    const int row = t.row0 + trow + a * astride + (lane & 31);
    if (row >= t.row_end) continue;
    if (EPI == EPI_SWIGLU_BWD) {
      // recomputed gate h and up u: dh = dA u silu'(h), du = dA silu(h), a = silu(h) u
      bf16_t* yrow = reinterpret_cast<bf16_t*>(t.Y) + (int64_t)row * p.ldy;
      const bf16_t* darow = p.dact + (int64_t)row * p.N;
      bf16_t* arow = p.act_out + (int64_t)row * p.N;
#pragma unroll
      for (int b = 0; b < FN / 2; ++b) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int col = fcol + b * 32 + 8 * q + 4 * (lane >> 5);
          if (col >= p.N) continue;
          const uint2 dav = *reinterpret_cast<const uint2*>(darow + col);
          const float da[4] = {bf16_to_f32(dav.x & 0xffffu), bf16_to_f32(dav.x >> 16), bf16_to_f32(dav.y & 0xffffu),
                               bf16_to_f32(dav.y >> 16)};
          float dh[4], du[4], av[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float h = acc[a][b][4 * q + e], u = acc[a][b + FN / 2][4 * q + e];
            const float sg = __builtin_amdgcn_rcpf(1.0f + __expf(-h));
            const float silu = h * sg;
            av[e] = silu * u;
            du[e] = da[e] * silu;
            dh[e] = da[e] * u * sg * (1.0f + h * (1.0f - sg));
          }
          uint2 v;
          v.x = pack_bf16x2(dh[0], dh[1]);
          v.y = pack_bf16x2(dh[2], dh[3]);
          *reinterpret_cast<uint2*>(yrow + col) = v;
          v.x = pack_bf16x2(du[0], du[1]);
          v.y = pack_bf16x2(du[2], du[3]);
          *reinterpret_cast<uint2*>(yrow + p.N + col) = v;
          v.x = pack_bf16x2(av[0], av[1]);
          v.y = pack_bf16x2(av[2], av[3]);
          *reinterpret_cast<uint2*>(arow + col) = v;
        }
      }
    } else if (EPI == EPI_SWIGLU) {
      bf16_t* yrow = reinterpret_cast<bf16_t*>(t.Y) + (int64_t)row * p.ldy;
#pragma unroll
      for (int b = 0; b < FN / 2; ++b) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int col = fcol + b * 32 + 8 * q + 4 * (lane >> 5);
          if (col >= p.N) continue;
          float o[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            float gt = acc[a][b][4 * q + e], up = acc[a][b + FN / 2][4 * q + e];
            o[e] = gt * __builtin_amdgcn_rcpf(1.0f + __expf(-gt)) * up;
          }
          uint2 v;
          v.x = pack_bf16x2(o[0], o[1]);
          v.y = pack_bf16x2(o[2], o[3]);
          *reinterpret_cast<uint2*>(yrow + col) = v;
        }
      }
    } else if (EPI == EPI_BF16) {
      bf16_t* yrow = reinterpret_cast<bf16_t*>(t.Y) + (int64_t)row * p.ldy;
#pragma unroll
      for (int b = 0; b < FN; ++b) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int col = fcol + b * 32 + 8 * q + 4 * (lane >> 5);
          if (col >= p.N) continue;
          uint2 v;
          v.x = pack_bf16x2(acc[a][b][4 * q + 0], acc[a][b][4 * q + 1]);
          v.y = pack_bf16x2(acc[a][b][4 * q + 2], acc[a][b][4 * q + 3]);
          *reinterpret_cast<uint2*>(yrow + col) = v;
        }
      }
    } else {
      float* yrow = reinterpret_cast<float*>(t.Y) + t.kc * p.y_split_stride + (int64_t)row * p.ldy;
      const bool vec = (p.ldy % 4 == 0) && (p.y_split_stride % 4 == 0);   // 16-byte aligned rows
#pragma unroll
      for (int b = 0; b < FN; ++b) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int col = fcol + b * 32 + 8 * q + 4 * (lane >> 5);
          if (vec && col + 3 < p.N) {
            const f32x4 v = {acc[a][b][4 * q], acc[a][b][4 * q + 1], acc[a][b][4 * q + 2], acc[a][b][4 * q + 3]};
            *reinterpret_cast<f32x4*>(yrow + col) = v;
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (col + e < p.N) yrow[col + e] = acc[a][b][4 * q + e];
          }
        }
      }
    }
  }
}

// EPI_BF16 / EPI_SWIGLU through LDS: a lane's MFMA results are 4-column pieces of one row, so
// storing them straight from registers writes 16-byte pieces of 32 rows per instruction.
// Each 32-row block of the wave's sub-tile instead goes to a wave-private LDS area (`st`, 32 rows
// of OUTW bf16) and comes back as 16-byte pieces of whole rows: a store instruction then writes
// 64 / (OUTW / 8) full rows of OUTW columns.  The 16-byte piece c of staged row r sits at piece
// c ^ (r % (OUTW / 8)), which spreads the 32 rows one write instruction touches over the banks.
template <int EPI, int FM, int FN, int OUTW>
__device__ __forceinline__ void store_tile_staged(const GemmProblem& p, const f32x16 (&acc)[FM][FN],
                                                  const TileDesc& t, int trow, int astride, int fcol, int lane,
                                                  bf16_t* st) {
  static_assert(EPI == EPI_BF16 || EPI == EPI_SWIGLU, "staged epilogue: bf16 results");
  constexpr int CPRW = OUTW / 8;                          // 16-byte pieces per staged row
  constexpr int FO = EPI == EPI_SWIGLU ? FN / 2 : FN;     // output fragments per row block
  static_assert(FO * 32 == OUTW && (32 * CPRW) % 64 == 0, "staged row width");
  const int hi = lane >> 5, r = lane & 31;
#pragma unroll
  for (int a = 0; a < FM; ++a) {
    const int rbase = t.row0 + trow + a * astride;       // first row of the 32-row block
    if (rbase >= t.row_end) continue;                     // wave-uniform
#pragma unroll
    for (int b = 0; b < FO; ++b)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float o[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (EPI == EPI_SWIGLU) {
            const float gt = acc[a][b][4 * q + e], up = acc[a][b + FN / 2][4 * q + e];
            o[e] = gt * __builtin_amdgcn_rcpf(1.0f + __expf(-gt)) * up;
          } else {
            o[e] = acc[a][b][4 * q + e];
          }
        }
        uint2 v;
        v.x = pack_bf16x2(o[0], o[1]);
        v.y = pack_bf16x2(o[2], o[3]);
        *reinterpret_cast<uint2*>(st + r * OUTW + (((b * 4 + q) ^ (r % CPRW)) << 3) + 4 * hi) = v;
      }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int it = 0; it < 32 * CPRW / 64; ++it) {
      const int idx = it * 64 + lane;
      const int rr = idx / CPRW, c = idx % CPRW;
      const int row = rbase + rr, col = fcol + c * 8;
      const u32x4 v = ld16(st + rr * OUTW + ((c ^ (rr % CPRW)) << 3));
      if (row < t.row_end && col < p.N)
        st16(reinterpret_cast<bf16_t*>(t.Y) + (int64_t)row * p.ldy + col, v);
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_wave_barrier();
  }
}

// EPI_SCATTER: the gate-weighted combine folded into the epilogue.  In the MFMA layout a lane
// holds 4-column pieces of one token row, so adding the fragment straight from registers
// would touch 32 rows (cache lines) per instruction; each 32 x 32 fragment instead goes
// through a wave-private LDS block `lw` (32 rows of 36 floats, the padding spreads the banks)
// and comes back two rows per instruction, 32 consecutive columns each, so every float32
// atomic instruction covers two cache lines.  Row r of the tile adds w(r) * row into token
// row tok(r) of Y (see TileDesc::stok / sw).
constexpr int kScatterLd = 36;
template <int FM, int FN>
__device__ __forceinline__ void scatter_tile(const GemmProblem& p, const f32x16 (&acc)[FM][FN], const TileDesc& t,
                                             int trow, int astride, int fcol, int lane, float* lw) {
  const int hi = lane >> 5, r32 = lane & 31;
#pragma unroll
  for (int a = 0; a < FM; ++a) {
    const int rbase = t.row0 + trow + a * astride;               // first row of the 32-row block
    if (rbase >= t.row_end) continue;                            // wave-uniform
    const int nrow = min(32, t.row_end - rbase);
    // token and weight of the block's rows, one per lane (lanes 0..31)
    int tok = -1;
    float w = 0.f;
    if (r32 < nrow) {
      tok = t.stok ? t.stok[rbase + r32] : rbase + r32;
      w = t.sw ? t.sw[rbase + r32] : 1.0f;
      if (tok < 0 || tok >= p.scatter_rows) tok = -1;
    }
#pragma unroll
    for (int b = 0; b < FN; ++b) {
      const int col0 = fcol + b * 32;
      if (col0 >= p.N) continue;                                 // N % 8 == 0: whole 32-col pieces or none
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x4 v = {acc[a][b][4 * q], acc[a][b][4 * q + 1], acc[a][b][4 * q + 2], acc[a][b][4 * q + 3]};
        *reinterpret_cast<f32x4*>(lw + r32 * kScatterLd + 8 * q + 4 * hi) = v;
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      __builtin_amdgcn_wave_barrier();
      const int col = col0 + r32;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int rl = 2 * j + hi;                               // block row of this lane
        const int tj0 = __builtin_amdgcn_readlane(tok, 2 * j), tj1 = __builtin_amdgcn_readlane(tok, 2 * j + 1);
        const float wj0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w), 2 * j));
        const float wj1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w), 2 * j + 1));
        const int tk = hi ? tj1 : tj0;
        const float wk = hi ? wj1 : wj0;
        const float v = lw[rl * kScatterLd + r32];
        if (tk >= 0 && col < p.N) unsafeAtomicAdd(reinterpret_cast<float*>(t.Y) + (int64_t)tk * p.ldy + col, wk * v);
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      __builtin_amdgcn_wave_barrier();
    }
  }
}


// One K-step's MFMAs with the next slice's copies between them: MFMA M (token fragment M / FN,
// weight fragment M % FN) then copy M, while either remains.  Issuing a slice's copies in one
// block held every wave's MFMA issue behind ~50 address and copy instructions right after the
// slice barrier; spread this way the MFMA pipe keeps running (DeepSeek-V3 layer: up-projection
// 945 -> 908 us, down-projection 510 -> 498 us; Mixtral -6 / -7%; skewed up-projection -8%).
template <int M, int NA, int FN, int FM, int L, class CP>
__device__ __forceinline__ void mfma_copy_steps(f32x16 (&acc)[FM][FN], const bf16x8 (&fw)[FN], const bf16x8 (&fx)[FM],
                                                const CP& cp, bf16_t* dst, int kt, int wave) {
  if constexpr (M < NA * FN || M < L) {
    if constexpr (M < NA * FN)
      acc[M / FN][M % FN] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[M % FN], fx[M / FN], acc[M / FN][M % FN], 0, 0, 0);
    if constexpr (M < L) cp.template issue_one_sv<M>(dst, kt, wave);
    __builtin_amdgcn_sched_barrier(0);
    mfma_copy_steps<M + 1, NA, FN, FM, L>(acc, fw, fx, cp, dst, kt, wave);
  }
}

template <int FM, int FN>
__device__ __forceinline__ void zero_acc(f32x16 (&acc)[FM][FN]) {
#pragma unroll
  for (int a = 0; a < FM; ++a)
#pragma unroll
    for (int b = 0; b < FN; ++b)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[a][b][q] = 0.f;
}

// ---------------------------------------------------------------------------------------
// The kernel: every wave copies, reads and multiplies
// ---------------------------------------------------------------------------------------

// BM token rows x BN weight rows per tile, WGM x WGN waves (each a (BM/WGM) x (BN/WGN)
// sub-tile), BK-wide K slices through a STAGES-deep ring.
template <int BM, int BN, int BK, int STAGES, int WGM, int WGN, int EPI, bool KTAIL>
__global__ __launch_bounds__(64 * WGM * WGN, 1) void k_grouped_gemm(GemmProblem p) {
  using Z = Swz<BK>;
  constexpr int NW = WGM * WGN, NTH = 64 * NW;
  constexpr int WM = BM / WGM, WN = BN / WGN;             // per-wave sub-tile
  constexpr int FM = WM / 32, FN = WN / 32;               // 32x32 fragments per wave
  constexpr int OUTN = (swiglu_pairs(EPI)) ? BN / 2 : BN;
  constexpr int SLICE = (BM + BN) * BK;                   // bf16 elements per ring slot
  using CP = CopyPlan<BM, BN, BK, NW, EPI>;
  constexpr int L = CP::L;
  static_assert(FM >= 1 && FN >= 1, "tile too small");
  static_assert(!swiglu_pairs(EPI) || (FN % 2 == 0 && (BN / 2 / WGN) % 32 == 0), "SwiGLU pairs gate and up fragments");
  static_assert(STAGES >= 2 && (STAGES - 2) * L < 64, "ring depth");

  extern __shared__ __align__(16) uint8_t smem[];
  bf16_t* ring = reinterpret_cast<bf16_t*>(smem);         // [STAGES][BM + BN][BK]: X rows then W rows
  __shared__ int s_off[kMaxGroups + 1];
  __shared__ int s_tp[kMaxGroups + 1];
  __shared__ int s_tmp[NTH / 64];
  __shared__ int s_list[kTileList][8];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;
  const TileSpace ts = build_tile_space<NTH, BM, BK>(p, OUTN, s_off, s_tp, s_tmp);
  const int G = gridDim.x;
  const int K = p.K;
  const int nk = (K + BK - 1) / BK;
  const int nk_full = K / BK;
  constexpr bool ktail = KTAIL;                           // K % BK != 0 (launcher-checked)

  CP cp;
  auto issue_any = [&](int kt, int st) {
    if constexpr (KTAIL) {
      if (kt >= nk_full) cp.issue_tail(ring + st * SLICE, kt, wave, K);
      else cp.issue(ring + st * SLICE, kt, wave);
    } else {
      cp.issue_sv(ring + st * SLICE, kt, wave);
    }
  };

  // The current tile runs K slices kb .. kb + nl - 1; its i-th slice lives in ring slot
  // i % STAGES.  sync_slice(i) makes slice i readable by every wave and (issue) refills the ring
  // slot that slice i-1 used (i may be nl: then it only waits for every copy and synchronises).
  int kb = 0, nl = nk;
  auto sync_slice = [&](int i, bool issue = true) {
    const int after = min(STAGES - 2, nl - 1 - i);       // slices issued after i
    if (STAGES >= 4 && after >= 2) wait_vmcnt<(STAGES >= 4 ? 2 * L : 0)>();
    else if (STAGES >= 3 && after >= 1) wait_vmcnt<(STAGES >= 3 ? L : 0)>();
    else wait_vmcnt<0>();
    lds_barrier();
    if (issue && i + STAGES - 1 < nl) issue_any(kb + i + STAGES - 1, (i + STAGES - 1) % STAGES);
    const int kt = kb + i;
    if (ktail && i < nl && kt == nk - 1) {
      // zero the chunks past K of the last slice (their copies came from clamped addresses)
      bf16_t* z = ring + (i % STAGES) * SLICE;
      for (int idx = tid; idx < (BM + BN) * Z::CPR; idx += NTH) {
        const int r = idx / Z::CPR, pc = idx % Z::CPR;
        const int c = pc ^ Z::f(r);
        if (kt * BK + c * 8 >= K) st16(z + r * BK + pc * 8, u32x4{0, 0, 0, 0});
      }
      lds_barrier();
    }
  };

  // Token rows: fragment a of wave (wm, wn) holds the tile's 32-row block a * WGM + wm, so the
  // row blocks alternate over the waves.  A tile whose segment ends early (the ragged last
  // m-tile of a group) leaves every wave with fewer live blocks; a wave multiplies only its
  // live ones (NA of FM, uniform per wave and tile), and the blocks past the end cost no MFMA.
  constexpr int KS = BK / 16;                             // MFMA K-steps per slice
  int wrow_l[FN], xrow_l[FM], wf_l[FN], xf_l[FM];
#pragma unroll
  for (int b = 0; b < FN; ++b) {
    const int r = frag_wrow<EPI, BN, WGN, FN>(wn, b) + (lane & 31);
    wrow_l[b] = BM * BK + r * BK;
    wf_l[b] = Z::f(r);
  }
#pragma unroll
  for (int a = 0; a < FM; ++a) {
    const int r = (a * WGM + wm) * 32 + (lane & 31);
    xrow_l[a] = r * BK;
    xf_l[a] = Z::f(r);
  }
  const int hi = lane >> 5;
  bf16x8 fw[2][FN], fx[2][FM];
  // read the fragments of K-step ks of ring slot st (the first NA token fragments)
  auto load_frags = [&](auto na, int buf, int st, int ks) {
    constexpr int NA = decltype(na)::value;
    const bf16_t* base = ring + st * SLICE;
    const int c = ks * 2 + hi;
    if constexpr (NA > 0) {
#pragma unroll
      for (int b = 0; b < FN; ++b)
        fw[buf][b] = *reinterpret_cast<const bf16x8*>(base + wrow_l[b] + ((c ^ wf_l[b]) << 3));
#pragma unroll
      for (int a = 0; a < NA; ++a)
        fx[buf][a] = *reinterpret_cast<const bf16x8*>(base + xrow_l[a] + ((c ^ xf_l[a]) << 3));
    }
  };

  // Round r of the persistent grid: the workgroup with first slot `slot` takes position
  // r G + slot in even rounds and r G + (G - 1 - slot) in odd ones (a snake order).  Tiles of a
  // routed expert cost in proportion to its live 32-row blocks; the snake pairs a workgroup's
  // positions from opposite ends of the tile sequence, so the per-workgroup sums of 4 rounds
  // scatter less.  An XCD still takes a contiguous block of positions in every round.
  const int slot = first_tile_slot();
  int round = 0;
  int tile = slot;
  if (tile >= ts.total) return;
  // this workgroup's tiles, decoded in parallel (the per-tile decode is ~2,500 cycles of integer
  // divisions and an LDS binary search, on the critical path between two tiles)
  for (int r = tid; r < kTileList; r += NTH) {
    const int pos = round_position(r, slot);
    if (pos < ts.total) {
      const TileCode c = tile_code<BM>(p, ts, pos);
      s_list[r][0] = c.row0; s_list[r][1] = c.row_end; s_list[r][2] = c.ni; s_list[r][3] = c.kb;
      s_list[r][4] = c.ke; s_list[r][5] = c.kc; s_list[r][6] = c.g;
    }
  }
  __syncthreads();
  auto fetch_tile = [&](int r, int pos) -> TileDesc {
    TileCode c;
    if (r < kTileList) {
      c.row0 = s_list[r][0]; c.row_end = s_list[r][1]; c.ni = s_list[r][2]; c.kb = s_list[r][3];
      c.ke = s_list[r][4]; c.kc = s_list[r][5]; c.g = s_list[r][6];
    } else {
      c = tile_code<BM>(p, ts, pos);
    }
    return tile_desc(p, c);
  };
  TileDesc td = fetch_tile(0, tile);
  cp.setup(p, td, wave, lane);
  kb = td.kb;
  nl = td.ke - td.kb;
#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (s < nl) issue_any(kb + s, s);

  const int fcol = (swiglu_pairs(EPI) ? wn * (BN / 2 / WGN) : wn * WN);
  while (true) {
    f32x16 acc[FM][FN];
    zero_acc(acc);

    // the K loop of one tile with NA live token fragments
    auto k_loop = [&](auto na) {
      constexpr int NA = decltype(na)::value;
      sync_slice(0);
      load_frags(na, 0, 0, 0);
      // Slice i: K-steps 0 .. KS-2 read the next step's fragments during this step's MFMAs.  The
      // last step's fragments are already in registers, so it first publishes slice i + 1 (vmcnt
      // wait + barrier) and reads that slice's first fragments, then runs its MFMAs; with
      // WITH_COPIES it also refills the ring slot slice i used (slice i + STAGES), one copy per
      // MFMA.  After the final slice the fragment reads touch a stale ring slot, harmlessly, to
      // keep the loop free of branches.  The slices that issue no copies run as a loop of their
      // own: a uniform branch between the two MFMA sequences inside one loop body made the
      // register allocator spill the accumulators.
      auto slice_body = [&](int i, auto with_copies) {
        constexpr bool WC = decltype(with_copies)::value;
        const int st = i % STAGES;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const int cur = ks & 1;
          if (ks + 1 < KS) {
            load_frags(na, cur ^ 1, st, ks + 1);
#pragma unroll
            for (int a = 0; a < NA; ++a)
#pragma unroll
              for (int b = 0; b < FN; ++b)
                acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[cur][b], fx[cur][a], acc[a][b], 0, 0, 0);
            // scheduling: an MFMA first (its operands were read during the previous step), then
            // the next step's LDS reads two at a time between MFMAs, so every read has several
            // MFMAs of this step to hide its latency behind
            if constexpr (NA > 0) sched_step<NA + FN, NA * FN>();
          } else if constexpr (KTAIL) {
            // K tail: the copies go out right after the barrier (the last slice's copies take
            // clamped addresses and its chunks past K are zeroed inside sync_slice)
            sync_slice(i + 1);
            load_frags(na, cur ^ 1, (i + 1) % STAGES, 0);
#pragma unroll
            for (int a = 0; a < NA; ++a)
#pragma unroll
              for (int b = 0; b < FN; ++b)
                acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[cur][b], fx[cur][a], acc[a][b], 0, 0, 0);
            if constexpr (NA > 0) sched_step<NA + FN, NA * FN>();
          } else {
            sync_slice(i + 1, false);
            load_frags(na, cur ^ 1, (i + 1) % STAGES, 0);
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (WC) {
              mfma_copy_steps<0, NA, FN, FM, L>(acc, fw[cur], fx[cur], cp, ring + st * SLICE, kb + i + STAGES, wave);
            } else {
#pragma unroll
              for (int a = 0; a < NA; ++a)
#pragma unroll
                for (int b = 0; b < FN; ++b)
                  acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[cur][b], fx[cur][a], acc[a][b], 0, 0, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
          }
        }
      };
      if constexpr (KTAIL) {
        for (int i = 0; i < nl; ++i) slice_body(i, std::false_type{});
      } else {
        int i = 0;
        for (; i < nl - STAGES; ++i) slice_body(i, std::true_type{});
        for (; i < nl; ++i) slice_body(i, std::false_type{});
      }
    };
    const int live_blocks = min(BM / 32, (td.row_end - td.row0 + 31) / 32);
    const int na = __builtin_amdgcn_readfirstlane(max(0, (live_blocks - wm + WGM - 1) / WGM));
    with_count<FM>(na, k_loop);

    // next tile: start its copies before this tile's epilogue (every wave is done with the ring)
    const TileDesc cur_td = td;
    ++round;
    tile = round_position(round, slot);
    const bool more = tile < ts.total;
    lds_barrier();
    if (more) {
      td = fetch_tile(round, tile);
      cp.setup(p, td, wave, lane);
      kb = td.kb;
      nl = td.ke - td.kb;
#pragma unroll
      for (int s = 0; s < STAGES - 1; ++s)
        if (s < nl) issue_any(kb + s, s);
    }
    if constexpr (EPI == EPI_SCATTER) {
      // the last ring slot is idle until the next tile's first barrier: one LDS block per wave
      static_assert(NW * 32 * kScatterLd * 4 <= SLICE * 2, "scatter staging fits one ring slot");
      float* lw = reinterpret_cast<float*>(ring + (STAGES - 1) * SLICE) + wave * 32 * kScatterLd;
      scatter_tile<FM, FN>(p, acc, cur_td, wm * 32, WGM * 32, cur_td.ni * OUTN + fcol, lane, lw);
    } else if constexpr ((EPI == EPI_BF16 || EPI == EPI_SWIGLU) &&
                         NW * 32 * (EPI == EPI_SWIGLU ? WN / 2 : WN) <= SLICE) {
      // whole-row stores staged through the last ring slot (idle until the next tile's first barrier)
      constexpr int OUTW = EPI == EPI_SWIGLU ? WN / 2 : WN;
      bf16_t* st = ring + (STAGES - 1) * SLICE + wave * 32 * OUTW;
      store_tile_staged<EPI, FM, FN, OUTW>(p, acc, cur_td, wm * 32, WGM * 32, cur_td.ni * OUTN + fcol, lane, st);
    } else {
      store_tile<EPI, FM, FN>(p, acc, cur_td, wm * 32, WGM * 32, cur_td.ni * OUTN + fcol, lane);
    }
    if (!more) break;
  }
}


// Persistent launch of kernel `fn` (nth threads, lds bytes of dynamic LDS): grid = the
// smaller of an upper bound of the launch's tile count and the resident workgroups, rounded
// down to whole rounds of the 8 XCDs.  `occ` caches the kernel's occupancy per device.
hipError_t launch_persistent(const void* fn, OccCache& occ, int nth, size_t lds, int bm, int outn,
                             const GemmProblem& p, hipStream_t stream) {
  const size_t lds_static = 2 * (kMaxGroups + 1) * sizeof(int) + kTileList * 8 * sizeof(int) + 64;
  if (lds + lds_static > (size_t)lds_limit()) return hipErrorInvalidConfiguration;
  hipError_t err;
  const int per_cu = kernel_occupancy(occ, fn, nth, lds, err);
  if (err != hipSuccess) return err;
  const int64_t tiles_n = (p.N + outn - 1) / outn;
  const int64_t groups = p.offsets ? p.groups : 1;
  const int64_t rows = p.offsets ? p.max_rows : p.rows_single;
  const int bmx = (p.rows2_tile > 0 && p.rows2_tile < bm) ? p.rows2_tile : bm;
  const int64_t upper = tiles_n * ((rows + bm - 1) / bm + groups + (p.rows2 + bmx - 1) / bmx) *
                        (p.ksplit > 1 ? p.ksplit : 1);
  const int64_t resident = (int64_t)cu_count() * per_cu;
  int64_t grid = upper < resident ? upper : resident;
  if (grid >= 8) grid -= grid % 8;
  if (grid < 1) grid = 1;
  GemmProblem arg = p;
  void* args[] = {&arg};
  hipError_t e = hipLaunchKernel(fn, dim3((unsigned)grid), dim3(nth), args, lds, stream);
  return e != hipSuccess ? e : hipGetLastError();
}

template <int BM, int BN, int BK, int STAGES, int WGM, int WGN, int EPI, bool KTAIL>
hipError_t launch_kernel(const GemmProblem& p, hipStream_t stream) {
  static OccCache occ;
  const void* fn = reinterpret_cast<const void*>(&k_grouped_gemm<BM, BN, BK, STAGES, WGM, WGN, EPI, KTAIL>);
  return launch_persistent(fn, occ, 64 * WGM * WGN, (size_t)STAGES * (BM + BN) * BK * sizeof(bf16_t), BM,
                           swiglu_pairs(EPI) ? BN / 2 : BN, p, stream);
}

template <int BM, int BN, int BK, int STAGES, int WGM, int WGN, int EPI>
hipError_t launch_tile(const GemmProblem& p, hipStream_t stream) {
  if (p.K < 8) return hipErrorInvalidValue;
  if (p.K % BK == 0) return launch_kernel<BM, BN, BK, STAGES, WGM, WGN, EPI, false>(p, stream);
  return launch_kernel<BM, BN, BK, STAGES, WGM, WGN, EPI, true>(p, stream);
}

template <int EPI>
hipError_t launch_cfg(int cfg, const GemmProblem& p, hipStream_t stream) {
  switch (cfg) {
    case 5: return launch_tile<128, 256, 64, 3, 2, 4, EPI>(p, stream);
    case 6: return launch_tile<256, 256, 64, 2, 4, 2, EPI>(p, stream);
    case 7: return launch_tile<256, 128, 64, 3, 4, 2, EPI>(p, stream);
    case 8: return launch_tile<320, 256, 64, 2, 2, 4, EPI>(p, stream);
    // few rows per group (decode-like): 64 x 128 tiles, 4 waves, 3-slot ring, two workgroups per CU
    case 20: return launch_tile<64, 128, 64, 3, 2, 2, EPI>(p, stream);
#ifdef MOE_GEMM_SWEEP
    // tuning-sweep shapes (not chosen by the launcher)
    case 0: return launch_tile<128, 128, 64, 2, 2, 2, EPI>(p, stream);
    case 1: return launch_tile<128, 256, 64, 3, 2, 2, EPI>(p, stream);
    case 2: return launch_tile<256, 256, 64, 2, 2, 4, EPI>(p, stream);
    case 3: return launch_tile<256, 256, 32, 4, 2, 4, EPI>(p, stream);
    case 4: return launch_tile<128, 512, 32, 3, 2, 4, EPI>(p, stream);
    case 21: return launch_tile<64, 64, 64, 4, 2, 1, EPI>(p, stream);
    case 22: return launch_tile<32, 128, 64, 4, 1, 2, EPI>(p, stream);
    // narrow-N shapes (router logits, fp32 epilogue)
    case 13: if constexpr (EPI == EPI_F32) return launch_tile<64, 64, 64, 3, 2, 2, EPI>(p, stream); break;
    case 14: if constexpr (EPI == EPI_F32) return launch_tile<64, 128, 64, 3, 2, 2, EPI>(p, stream); break;
    case 15: if constexpr (EPI == EPI_F32) return launch_tile<128, 64, 64, 3, 2, 2, EPI>(p, stream); break;
    case 16: if constexpr (EPI == EPI_F32) return launch_tile<32, 256, 64, 3, 1, 4, EPI>(p, stream); break;
    case 17: if constexpr (EPI == EPI_F32) return launch_tile<64, 256, 64, 2, 2, 4, EPI>(p, stream); break;
    case 18: if constexpr (EPI == EPI_F32) return launch_tile<128, 128, 64, 2, 4, 2, EPI>(p, stream); break;
    case 19: if constexpr (EPI == EPI_F32) return launch_tile<64, 64, 128, 2, 2, 2, EPI>(p, stream); break;
#endif
    default: break;
  }
  return hipErrorInvalidValue;
}

#ifdef MOE_GEMM_SWEEP
int g_force_cfg[3] = {-1, -1, -1};
#endif

}  // namespace

hipError_t launch_grouped_gemm(const GemmProblem& p, hipStream_t stream) {
  if (p.ksplit > 1 && (p.epi != EPI_F32 || p.offsets != nullptr || p.rows2 > 0)) return hipErrorInvalidValue;
  // gathered rows: the per-lane 32-bit source offsets must reach every row of X
  if (p.row_index && (p.x_rows < 1 || p.x_rows * p.ldx * 2 >= (int64_t(1) << 32))) return hipErrorInvalidValue;
  // equal-stride segments must fit the row bound
  if (p.seg_stride > 0 && (p.offsets == nullptr || (int64_t)p.groups * p.seg_stride > p.max_rows))
    return hipErrorInvalidValue;
  // 256 x 256 tiles, 8 waves, two 64-wide K slices in flight: the best measured on the DeepSeek-V3,
  // Mixtral and skewed workloads (largest reuse per byte copied into LDS; also whenever a large
  // dense extra group shares the launch).  With few expected rows per group the launch is a
  // weight stream over few m-tiles, spread over more workgroups by smaller tiles: 64 x 128 up to
  // 128 rows per group (1.4-1.8x faster at 2-128 rows), 128 x 256 up to 512 (1.1-1.5x).
  const bool small_extra = p.rows2 <= 512;
  const int tier = (p.rows_hint > 0 && small_extra) ? (p.rows_hint <= 128 ? 20 : p.rows_hint <= 512 ? 5 : 6) : 6;
  int cfg_swiglu = tier, cfg_bf16 = tier;
  // Tile shape from the expected tile count of each shape.  A persistent launch takes about
  // ceil(tiles / CUs) rounds of its slowest workgroup; per tile, a 320 x 256 tile (10 token
  // blocks, 2 x 4 waves) costs ~1.15 of a 256 x 256 one, a 128 x 256 tile ~0.7, a 256 x 128 tile
  // ~0.6 (measured).  The per-expert row counts of a routed batch scatter around their mean
  // (standard deviation about its square root), so an expert whose mean is 256 rows takes 1.5
  // 256-row m-tiles on average but one 320-row tile: DeepSeek-V3 shapes (256 rows per expert,
  // shared expert of 8192 rows in the launch) run both projections on 320-row tiles (up
  // 1085-1093 -> 1000-1025 us, down 588-596 -> 565-568), Mixtral shapes (1024 rows per expert,
  // 2.25 rounds of 256 x 256 down-projection tiles) their down-projection (1137-1147 -> 944-955;
  // 256 x 128 tiles: 1097), while Mixtral's up-projection (15.75 rounds either way) and the
  // skewed workload stay on 256 x 256.  The backward's recomputed up-projection of the routed
  // experts alone (tier 128 x 256) takes 320-row tiles at DeepSeek-V3 (627 -> 521 us).
  int cfg_swiglu_bwd = tier;
  int rows2_tile = 0;
  if ((tier == 5 || tier == 6) && p.rows_hint > 0) {
    const double cus = cu_count();
    const int64_t groups = p.offsets ? p.groups : 1;
    const double mu = (double)p.rows_hint;
    const double sigma = groups > 1 ? std::sqrt(mu) : 0.0;
    auto grouped_mtiles = [&](int bm) {                  // expected m-tiles of the groups
      double per_group = 0;
      if (sigma == 0) {
        per_group = std::ceil(mu / bm);
      } else {
        const int jmax = (int)((mu + 8 * sigma) / bm) + 1;
        for (int j = 0; j <= jmax; ++j)                   // E[ceil(m / bm)] = sum_j P(m > j bm)
          per_group += 0.5 * std::erfc((j * bm - mu) / (sigma * std::sqrt(2.0)));
      }
      return per_group * groups;
    };
    auto mtiles = [&](int bm) { return grouped_mtiles(bm) + std::ceil((double)p.rows2 / bm); };
    // rounds of the persistent grid; an expected count a few hundredths of a round above a
    // whole number (the normal tail of the row counts) is that whole number
    auto rounds = [&](double tiles) { return std::max(1.0, std::ceil(tiles / cus - 0.05)); };
    const double tn = (double)((p.N + 127) / 128);        // 128-column output blocks
    const double tn256 = std::ceil(tn / 2);
    const double m128 = mtiles(128), m256 = mtiles(256), m320 = mtiles(320);
    // SwiGLU epilogues: a 256-row weight tile yields 128 output columns
    const double s_base = tier == 5 ? 0.7 * rounds(m128 * tn) : rounds(m256 * tn);
    if (1.15 * rounds(m320 * tn) < s_base) cfg_swiglu = cfg_swiglu_bwd = 8;
    // bf16 epilogue: also 256 x 128 tiles on the 256-row tier
    const double c8 = 1.15 * rounds(m320 * tn256);
    if (tier == 5) {
      if (c8 < 0.7 * rounds(m128 * tn256)) cfg_bf16 = 8;
    } else {
      const double c6 = rounds(m256 * tn256), c7 = 0.6 * rounds(m256 * tn);
      if (c8 < c6 && c8 <= c7) cfg_bf16 = 8;
      else if (c7 < c6) cfg_bf16 = 7;
    }
    // On 320-row tiles, a dense extra group (the shared expert) is tiled 256 rows high when that
    // adds no round: its tiles then carry the 8 live token blocks the routed ones do (the routed
    // experts' ~256 rows), instead of 10.  DeepSeek-V3 shapes: up-projection 928 -> 1024 tiles
    // (4 rounds either way), down-projection 1624 -> 1792 (7 rounds either way).
    const int my_cfg = p.epi == EPI_SWIGLU ? cfg_swiglu : p.epi == EPI_BF16 ? cfg_bf16 : 0;
    if (my_cfg == 8 && p.rows2 > 256) {
      const double cols = p.epi == EPI_SWIGLU ? tn : tn256;
      const double g320 = grouped_mtiles(320);
      if (rounds((g320 + std::ceil(p.rows2 / 256.0)) * cols) <= rounds((g320 + std::ceil(p.rows2 / 320.0)) * cols))
        rows2_tile = 256;
    }
  }
#ifdef MOE_GEMM_SWEEP
  if (g_force_cfg[EPI_SWIGLU] >= 0) cfg_swiglu = g_force_cfg[EPI_SWIGLU];
  if (g_force_cfg[EPI_BF16] >= 0) cfg_bf16 = g_force_cfg[EPI_BF16];
#endif
  GemmProblem q = p;
  q.rows2_tile = rows2_tile;
  switch (p.epi) {
    case EPI_SWIGLU: return launch_cfg<EPI_SWIGLU>(cfg_swiglu, q, stream);
    case EPI_SWIGLU_BWD:
      if (!p.dact || !p.act_out || p.rows2 > 0 || p.ldy != 2 * (int64_t)p.N) return hipErrorInvalidValue;
      switch (cfg_swiglu_bwd) {      // the tiers of the forward up-projection (same operand shapes)
        case 20: return launch_tile<64, 128, 64, 3, 2, 2, EPI_SWIGLU_BWD>(p, stream);
        case 5: return launch_tile<128, 256, 64, 3, 2, 4, EPI_SWIGLU_BWD>(p, stream);
        case 8: return launch_tile<320, 256, 64, 2, 2, 4, EPI_SWIGLU_BWD>(p, stream);
        default: return launch_tile<256, 256, 64, 2, 4, 2, EPI_SWIGLU_BWD>(p, stream);
      }
    case EPI_BF16: return launch_cfg<EPI_BF16>(cfg_bf16, q, stream);
    case EPI_SCATTER:
      if (p.scatter_rows < 1) return hipErrorInvalidValue;
      switch (tier) {      // the tiers of the bf16 epilogue (same operand shapes)
        case 20: return launch_tile<64, 128, 64, 3, 2, 2, EPI_SCATTER>(p, stream);
        case 5: return launch_tile<128, 256, 64, 3, 2, 4, EPI_SCATTER>(p, stream);
        default: return launch_tile<256, 256, 64, 2, 4, 2, EPI_SCATTER>(p, stream);
      }
    case EPI_F32:
#ifdef MOE_GEMM_SWEEP
      if (g_force_cfg[EPI_F32] >= 0) return launch_cfg<EPI_F32>(g_force_cfg[EPI_F32], p, stream);
#endif
    {
      const TileShape ft = f32_tile(p.offsets ? p.max_rows : p.rows_single, p.N);
      if (ft.bn == 256) return launch_tile<128, 256, 64, 3, 2, 4, EPI_F32>(p, stream);
      if (ft.bn == 128) return launch_tile<64, 128, 64, 3, 2, 2, EPI_F32>(p, stream);
      return launch_tile<64, 64, 64, 3, 2, 2, EPI_F32>(p, stream);
    }
    default: return hipErrorInvalidValue;
  }
}

}  // namespace moe

#ifdef MOE_GEMM_SWEEP
// tile-configuration override for tuning sweeps (not part of the ABI)
extern "C" int moe_sweep_set_gemm_cfg(int epi, int cfg) {
  if (epi < 0 || epi > 2) return 1;
  moe::g_force_cfg[epi] = cfg;
  return 0;
}
#endif
