// Grouped GEMMs of the expert-MLP backward on gfx950 bf16 MFMA (v_mfma_f32_32x32x16_bf16),
// fp32 accumulation, bf16 results.
//
//   Y[m, n] = sum_k X[m, k] * W[n, k]
//
// The backward of the SwiGLU expert MLP (the dual GEMMs in transposed layout of the paper's
// training leg, Section 4, engine registration) needs operands whose reduction index is
// not the contiguous one:
//   dA  = dY W2          W2 is stored [d][F]: the weight operand is MN-major
//   dX  = [dH dU] w13    w13 is stored [2F][d]: the weight operand is MN-major
//   dW2 = dY^T A         both operands are row-major activations reduced over their rows
//   dW13 = [dH dU]^T X   (k = the expert's rows): both MN-major, one output per expert
// Each operand therefore has one of two LDS layouts:
//   K-major  [R][BK], 16-byte chunk c of row r at chunk c ^ f(r) (the forward's swizzle),
//            fragments by ds_read_b128 (8 consecutive k of one row per lane);
//   MN-major [BK][R], chunk c of k-row k at chunk c ^ g(k), g(k) = (k & 3) << 2, fragments
//            by two ds_read_b64_tr_b16 (the gfx950 transpose read).  Within each 16-lane
//            group that instruction hands lane i element (i & 3) of the 8-byte pieces the
//            group's lanes 4 j + (i >> 2) (j = 0..3) point at; when lane 4 j + q of group G
//            points at k-row K + 8 (G >> 1) + 4 h + j, columns m0 + 16 (G & 1) + 4 q .. + 3,
//            lane l receives column m0 + (l & 31) at k = K + 8 (l >> 5) + 4 h + 0..3: the
//            MFMA operand layout.  Those eight pieces cover k-rows K..K+3 and K+8..K+11, 64
//            bytes each, and g(k) puts the four rows of each half in different 64-byte
//            quarters of a 256-byte bank cycle (g only depends on k & 3 = j, so it is a
//            per-lane constant).
// Both layouts are filled by the direct-to-LDS 16-byte copies (lane i of a wave instruction
// writes bytes [16 i, 16 i + 16) of a 1 KB block; the swizzle picks the global chunk).
//
// Two groupings (see GemmBwdProblem): row segments (dA, dX: group g's rows of X and Y, its
// own weights) and K segments (dW: group g reduces over its rows, one M x N output each).
// Persistent workgroups walk the tile list; the next tile's first slice is in flight during
// the epilogue.  K tails (segments of any length) are fetched from clamped addresses and
// zeroed in LDS; rows / columns past the edges are clamped and never stored.
#include <algorithm>
#include <cmath>
#include <type_traits>

#include "common.hpp"
#include "gemm_device.hpp"
#include "kernels.hpp"

namespace moe {
namespace {

typedef short v4s __attribute__((ext_vector_type(4)));
typedef short v8s __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) v4s lds_v4s;

__device__ __forceinline__ bf16x8 tr_pair(const bf16_t* p0, const bf16_t* p1) {
  const v4s a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(p0));
  const v4s b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(p1));
  const v8s c = __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, c);
}

// One tile: output rows [m0, m_end) x columns [n0, N) of group g, K range [kbeg, kbeg + klen).
struct BTile {
  int g, m0, m_end, n0, kbeg, klen;
};

// Copies of one operand's slice (R tile rows x BK) into its LDS block, over NW waves.
// MN = false: global (r, k) at base + r * ld + k; MN = true: global (k, r) at base + k * ld + r.
template <int R, int BK, int NW, bool MN>
struct OpCopy {
  static constexpr int CH = R * BK / 8;                  // 16-byte chunks per slice
  static constexpr int L = CH / 64 / NW;                 // wave instructions per slice and wave
  static_assert(CH % (64 * NW) == 0 && L >= 1, "operand tile too small for the waves");
  static constexpr int CPR = MN ? R / 8 : BK / 8;        // chunks per LDS row
  static_assert(!MN || CPR >= 16, "MN-major tiles need >= 128 elements per k-row");
  using Z = Swz<BK>;

  const char* base;        // element (0, 0) of the tile's K range
  int64_t ld2;             // row stride in bytes
  uint32_t off[L];         // per lane: byte offset inside a slice

  // rlast: last valid tile row (K-major) / last valid 8-column chunk start (MN-major)
  __device__ __forceinline__ void setup(const bf16_t* b, int64_t ld, int rlast, int wave, int lane) {
    base = reinterpret_cast<const char*>(b);
    ld2 = ld * 2;
#pragma unroll
    for (int j = 0; j < L; ++j) {
      const int cid = (wave + NW * j) * 64 + lane;
      const int row = cid / CPR, pc = cid % CPR;
      if constexpr (MN) {
        const int lc = pc ^ ((row & 3) << 2);
        off[j] = (uint32_t)(row * ld2 + min(lc * 8, rlast) * 2);
      } else {
        const int lc = pc ^ Z::f(row);
        off[j] = (uint32_t)(min(row, rlast) * ld2 + lc * 16);
      }
    }
  }

  // k offset inside the slice of the lane's chunk in instruction j: its k-row (MN-major) or
  // the first k of its chunk (K-major); recomputed for the tail slice only
  __device__ __forceinline__ static int chunk_k(int j, int wave, int lane) {
    if constexpr (MN && 64 % CPR == 0) {
      // the instruction's first k-row is wave-uniform; a lane adds lane / CPR
      return (wave + NW * j) * (64 / CPR) + lane / CPR;
    } else {
      const int cid = (wave + NW * j) * 64 + lane;
      const int row = cid / CPR, pc = cid % CPR;
      if constexpr (MN) return row;
      else return (pc ^ Z::f(row)) * 8;
    }
  }

  // slice kt of a K range of klen into the LDS block dst (this wave's L instructions); KT =
  // false: klen is a multiple of BK (no tail slice, no tail code)
  template <bool KT>
  __device__ __forceinline__ void issue(bf16_t* dst, int kt, int klen, int wave) const {
    const int lane = threadIdx.x & 63;
    const int k0 = kt * BK;
    const bool tail = KT && k0 + BK > klen;
    const char* sb = MN ? base + (int64_t)k0 * ld2 : base + k0 * 2;
#pragma unroll
    for (int j = 0; j < L; ++j) {
      uint32_t o = off[j];
      if (tail) {
        const int kr = chunk_k(j, wave, lane);
        if constexpr (MN) o -= (uint32_t)(max(k0 + kr - (klen - 1), 0) * ld2);
        else o -= (uint32_t)(max(k0 + kr - (klen - 8), 0) * 2);
      }
      dma16_sv(sb, o, dst + (wave + NW * j) * 512);
    }
  }

  // zero the parts of slice kt past klen (after it landed)
  __device__ __forceinline__ static void zero_tail(bf16_t* blk, int kt, int klen, int tid, int nth) {
    const int k0 = kt * BK;
    for (int c = tid; c < CH; c += nth) {
      const int row = c / CPR, pc = c % CPR;
      bool dead;
      if constexpr (MN) dead = k0 + row >= klen;
      else dead = k0 + ((pc ^ Z::f(row)) * 8) >= klen;
      if (dead) st16(blk + c * 8, u32x4{0, 0, 0, 0});
    }
  }
};

template <int BM, int BN, int BK, int STAGES, int WGM, int WGN, bool XMN, bool WMN, int MODE, int OCC, bool KTAIL>
__global__ __launch_bounds__(64 * WGM * WGN, OCC) void k_gemm_bwd(GemmBwdProblem p) {
  constexpr int NW = WGM * WGN, NTH = 64 * NW;
  static_assert(STAGES >= 2 && STAGES <= 4, "ring depth");
  constexpr int WM = BM / WGM, WN = BN / WGN, FM = WM / 32, FN = WN / 32;
  constexpr int KS = BK / 16;
  constexpr int SLICE = (BM + BN) * BK;
  static_assert(FM >= 1 && FN >= 1, "wave tile");
  static_assert(MODE == BWD_KSEG || !XMN, "row segments take a K-major X");
  static_assert(NW * 32 * WN <= SLICE, "epilogue staging fits one ring slot");
  static_assert((32 * (WN / 8)) % 64 == 0, "epilogue pieces per wave");
  using CX = OpCopy<BM, BK, NW, XMN>;
  using CW = OpCopy<BN, BK, NW, WMN>;
  using Z = Swz<BK>;

  extern __shared__ __align__(16) uint8_t smem[];
  bf16_t* ring = reinterpret_cast<bf16_t*>(smem);        // [STAGES][X block | W block]
  __shared__ int s_off[kMaxGroups];                      // first row of each group
  __shared__ int s_len[kMaxGroups];                      // rows of each group
  __shared__ int s_tp[MODE == BWD_ROWS ? kMaxGroups + 1 : 1];   // row segments: first tile of each group
  __shared__ int s_tmp[NW];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;
  const int groups = p.groups;
  const int tn = (p.N + BN - 1) / BN;

  // segment table: begin / length of every group (clamped to the row bound)
  const int cap = (int)p.max_rows;
  for (int g = tid; g < groups; g += NTH) {
    int b, e;
    if (p.seg_stride > 0) {
      b = g * p.seg_stride;
      e = b + min(max(p.offsets[g], 0), p.seg_stride);
    } else {
      b = min(max(p.offsets[g], 0), cap);
      e = min(max(p.offsets[g + 1], b), cap);
    }
    s_off[g] = b;
    s_len[g] = e - b;
  }
  __syncthreads();
  int total;
  if constexpr (MODE == BWD_ROWS) {
    // tiles per group = ceil(len / BM) * tn, prefix-summed into s_tp (first tile of g)
    constexpr int PER = (kMaxGroups + NTH - 1) / NTH;
    int loc[PER], lsum = 0;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int g = tid * PER + i;
      loc[i] = g < groups ? ((s_len[g] + BM - 1) / BM) * tn : 0;
      lsum += loc[i];
    }
    int excl;
    total = block_exclusive_scan<NTH>(lsum, s_tmp, excl);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int g = tid * PER + i;
      if (g < groups) s_tp[g] = excl;
      excl += loc[i];
    }
    if (tid == 0) s_tp[groups] = total;
    __syncthreads();
  } else {
    total = groups * ((p.M + BM - 1) / BM) * tn;
  }

  auto decode = [&](int tile) -> BTile {
    BTile t;
    if constexpr (MODE == BWD_ROWS) {
      int lo = 0, hi = groups;
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (s_tp[mid] <= tile) lo = mid; else hi = mid;
      }
      t.g = __builtin_amdgcn_readfirstlane(lo);
      const int local = tile - __builtin_amdgcn_readfirstlane(s_tp[t.g]);
      const int len = __builtin_amdgcn_readfirstlane(s_len[t.g]);
      const int tm = (len + BM - 1) / BM;
      const int mi = local % tm, ni = local / tm;         // m-fastest: tiles of one weight panel adjacent
      const int b = __builtin_amdgcn_readfirstlane(s_off[t.g]);
      t.m0 = b + mi * BM;
      t.m_end = b + len;
      t.n0 = ni * BN;
      t.kbeg = 0;
      t.klen = p.K;
    } else {
      const int tm = (p.M + BM - 1) / BM;
      t.g = tile / (tm * tn);
      const int local = tile - t.g * tm * tn;
      t.m0 = (local % tm) * BM;
      t.m_end = p.M;
      t.n0 = (local / tm) * BN;
      t.kbeg = __builtin_amdgcn_readfirstlane(s_off[t.g]);
      t.klen = __builtin_amdgcn_readfirstlane(s_len[t.g]);
    }
    return t;
  };

  CX cx;
  CW cw;
  auto setup = [&](const BTile& t) {
    // X operand: K-major rows [m0, m_end) of X (row segments), or MN-major columns of the
    // group's rows (K segments)
    if constexpr (XMN) cx.setup(p.X + (int64_t)t.kbeg * p.ldx + t.m0, p.ldx, t.m_end - 8 - t.m0, wave, lane);
    else cx.setup(p.X + (int64_t)t.m0 * p.ldx + t.kbeg, p.ldx, t.m_end - 1 - t.m0, wave, lane);
    const bf16_t* wg = MODE == BWD_ROWS ? p.W + (int64_t)t.g * p.w_group_stride : p.W;
    if constexpr (WMN) cw.setup(wg + (int64_t)t.kbeg * p.ldw + t.n0, p.ldw, p.N - 8 - t.n0, wave, lane);
    else cw.setup(wg + (int64_t)t.n0 * p.ldw + t.kbeg, p.ldw, p.N - 1 - t.n0, wave, lane);
  };
  auto issue = [&](int kt, int slot, int klen) {
    bf16_t* dst = ring + slot * SLICE;
    cx.template issue<KTAIL>(dst, kt, klen, wave);
    cw.template issue<KTAIL>(dst + BM * BK, kt, klen, wave);
  };

  // per-lane LDS fragment offsets (elements), K-step 0
  int xo[FM][2], wo[FN][2];
  {
    const int hi = lane >> 5, j = (lane >> 2) & 3, q = lane & 3, g1 = (lane >> 4) & 1;
#pragma unroll
    for (int a = 0; a < FM; ++a) {
      const int blk = a * WGM + wm;                       // 32-row block of the tile
      if constexpr (XMN) {
        const int lc = blk * 4 + 2 * g1 + (q >> 1);
        xo[a][0] = (8 * hi + j) * BM + ((lc ^ (j << 2)) << 3) + (q & 1) * 4;   // h = 1: + 4 BM
        xo[a][1] = 0;
      } else {
        const int r = blk * 32 + (lane & 31);
        xo[a][0] = r * BK;
        xo[a][1] = Z::f(r);
      }
    }
#pragma unroll
    for (int b = 0; b < FN; ++b) {
      const int blk = wn * FN + b;
      if constexpr (WMN) {
        const int lc = blk * 4 + 2 * g1 + (q >> 1);
        wo[b][0] = (8 * hi + j) * BN + ((lc ^ (j << 2)) << 3) + (q & 1) * 4;   // h = 1: + 4 BN
        wo[b][1] = 0;
      } else {
        const int r = blk * 32 + (lane & 31);
        wo[b][0] = r * BK;
        wo[b][1] = Z::f(r);
      }
    }
  }
  const int hi = lane >> 5;
  auto frag_x = [&](const bf16_t* blk, int a, int ks) -> bf16x8 {
    if constexpr (XMN) return tr_pair(blk + ks * 16 * BM + xo[a][0], blk + ks * 16 * BM + 4 * BM + xo[a][0]);
    else return *reinterpret_cast<const bf16x8*>(blk + xo[a][0] + (((ks * 2 + hi) ^ xo[a][1]) << 3));
  };
  auto frag_w = [&](const bf16_t* blk, int b, int ks) -> bf16x8 {
    if constexpr (WMN) return tr_pair(blk + ks * 16 * BN + wo[b][0], blk + ks * 16 * BN + 4 * BN + wo[b][0]);
    else return *reinterpret_cast<const bf16x8*>(blk + wo[b][0] + (((ks * 2 + hi) ^ wo[b][1]) << 3));
  };

  int tile = first_tile_slot();
  if (tile >= total) return;
  const int G = gridDim.x;
  BTile td = decode(tile);
  setup(td);
  int nl = (td.klen + BK - 1) / BK;
#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (s < nl) issue(s, s, td.klen);

  // sync_slice(i): slice i landed for every wave and every wave is done reading slice i - 1's
  // slot, which then takes slice i + STAGES - 1 (a partial last slice is zeroed past the K
  // range).  Slices issued after slice i may stay in flight, except on a tile's first slice:
  // the previous tile's result stores are queued behind its copies then, and loads and stores
  // are not assumed to complete in order, so everything is drained.
  constexpr int L = CX::L + CW::L;                       // copy instructions per slice and wave
  auto sync_slice = [&](int i) {
    const int after = min(STAGES - 2, nl - 1 - i);
    if (STAGES >= 4 && i > 0 && after >= 2) wait_vmcnt<(STAGES >= 4 ? 2 * L : 0)>();
    else if (STAGES >= 3 && i > 0 && after >= 1) wait_vmcnt<(STAGES >= 3 ? L : 0)>();
    else wait_vmcnt<0>();
    lds_barrier();
    if (i + STAGES - 1 < nl) issue(i + STAGES - 1, (i + STAGES - 1) % STAGES, td.klen);
    if (KTAIL && i < nl && (i + 1) * BK > td.klen) {
      bf16_t* xs = ring + (i % STAGES) * SLICE;
      CX::zero_tail(xs, i, td.klen, tid, NTH);
      CW::zero_tail(xs + BM * BK, i, td.klen, tid, NTH);
      lds_barrier();
    }
  };
  bf16x8 fx[2][FM], fw[2][FN];
  // the first NA token fragments (the live ones) and every weight fragment of K-step ks
  auto load_frags = [&](auto na, int buf, const bf16_t* xs, int ks) {
    constexpr int NA = decltype(na)::value;
#pragma unroll
    for (int a = 0; a < NA; ++a) fx[buf][a] = frag_x(xs, a, ks);
#pragma unroll
    for (int b = 0; b < FN; ++b) fw[buf][b] = frag_w(xs + BM * BK, b, ks);
  };

  while (true) {
    f32x16 acc[FM][FN];
#pragma unroll
    for (int a = 0; a < FM; ++a)
#pragma unroll
      for (int b = 0; b < FN; ++b)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.f;

    // the K loop with NA live token blocks for this wave: the tile's 32-row blocks alternate over
    // the waves (block a * WGM + wm), and blocks past the segment's end (the ragged last m-tile
    // of a group) cost no MFMA; every wave still copies and meets every barrier
    auto k_loop = [&](auto na) {
      constexpr int NA = decltype(na)::value;
      if (nl == 0) return;
      sync_slice(0);
      if constexpr (NA > 0) load_frags(na, 0, ring, 0);
      for (int i = 0; i < nl; ++i) {
        const bf16_t* xs = ring + (i % STAGES) * SLICE;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const int cur = ks & 1;
          if (ks + 1 < KS) {
            if constexpr (NA > 0) load_frags(na, cur ^ 1, xs, ks + 1);
          } else {
            // this step's operands are in registers: publish the next slice now, so the barrier
            // and its first reads overlap this step's MFMAs (after the last slice the reads hit
            // a stale slot, harmlessly)
            sync_slice(i + 1);
            if constexpr (NA > 0) load_frags(na, cur ^ 1, ring + ((i + 1) % STAGES) * SLICE, 0);
          }
          if constexpr (NA > 0) {
#pragma unroll
            for (int a = 0; a < NA; ++a)
#pragma unroll
              for (int b = 0; b < FN; ++b)
                acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[cur][b], fx[cur][a], acc[a][b], 0, 0, 0);
            sched_step<NA * (XMN ? 2 : 1) + FN * (WMN ? 2 : 1), NA * FN>();
          }
        }
      }
    };
    const int live_blocks = min(BM / 32, (td.m_end - td.m0 + 31) / 32);
    const int na = __builtin_amdgcn_readfirstlane(max(0, (live_blocks - wm + WGM - 1) / WGM));
    // weight-gradient tiles are full except at the edge of M: every block is computed there (the
    // dead rows are clamped copies and are not stored), which leaves one K loop in the kernel
    if constexpr (MODE == BWD_KSEG) k_loop(std::integral_constant<int, FM>{});
    else with_count<FM>(na, k_loop);

    // next tile's first slice goes into slot 0 once every wave is done reading the ring
    const BTile cur = td;
    tile += G;
    const bool more = tile < total;
    wait_vmcnt<0>();
    lds_barrier();
    if (more) {
      td = decode(tile);
      setup(td);
      nl = (td.klen + BK - 1) / BK;
#pragma unroll
      for (int s = 0; s < STAGES - 1; ++s)
        if (s < nl) issue(s, s, td.klen);
    }

    if (MODE == BWD_KSEG && p.Yf) {
      // float32 results straight from the accumulators: lane holds 4 consecutive columns of one row
      float* yf = p.Yf + (int64_t)cur.g * p.y_group_stride;
#pragma unroll
      for (int a = 0; a < FM; ++a) {
        const int row = cur.m0 + (a * WGM + wm) * 32 + (lane & 31);
        if (row >= cur.m_end) continue;
#pragma unroll
        for (int b = 0; b < FN; ++b)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int col = cur.n0 + wn * WN + b * 32 + 8 * q + 4 * hi;
            const f32x4 v = {acc[a][b][4 * q], acc[a][b][4 * q + 1], acc[a][b][4 * q + 2], acc[a][b][4 * q + 3]};
            if (col < p.N) *reinterpret_cast<f32x4*>(yf + (int64_t)row * p.ldy + col) = v;
          }
      }
      if (!more) break;
      continue;
    }
    // epilogue, one 32-row block at a time through this wave's area of the idle last ring slot:
    // the lane's 4-column pieces (row lane & 31, columns 32 b + 8 q + 4 hi) go to LDS, then
    // every lane stores 16-byte pieces of whole rows (WN columns each), so a store instruction
    // writes full cache lines of 64 / (WN / 8) rows.  The 16-byte piece c of staged row r sits
    // at piece c ^ (r % (WN / 8)), spreading the 32 rows a write instruction touches over the
    // banks.
    bf16_t* yg = p.Y + (MODE == BWD_KSEG ? (int64_t)cur.g * p.y_group_stride : 0);
    bf16_t* st_area = ring + (STAGES - 1) * SLICE + wave * 32 * WN;
    constexpr int CPRW = WN / 8;                          // 16-byte pieces per staged row
#pragma unroll
    for (int a = 0; a < FM; ++a) {
      const int rbase = cur.m0 + (a * WGM + wm) * 32;
      if (rbase >= cur.m_end) continue;                   // wave-uniform
#pragma unroll
      for (int b = 0; b < FN; ++b)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          uint2 v;
          v.x = pack_bf16x2(acc[a][b][4 * q + 0], acc[a][b][4 * q + 1]);
          v.y = pack_bf16x2(acc[a][b][4 * q + 2], acc[a][b][4 * q + 3]);
          const int r = lane & 31;
          *reinterpret_cast<uint2*>(st_area + r * WN + (((b * 4 + q) ^ (r % CPRW)) << 3) + 4 * hi) = v;
        }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      __builtin_amdgcn_wave_barrier();
      // unrolled by 4, not fully: fully unrolled, the eight per-lane staging addresses were
      // hoisted out of the tile loop and spilled, and every store then reloaded one behind an
      // s_waitcnt vmcnt(0) that also waited for the next tile's slice copies and the previous
      // stores (32 experts of 256 rows, d = 7168, F = 2048: dW13 992 -> 893 us, dW2 499 -> 454)
#pragma unroll 4
      for (int it = 0; it < 32 * CPRW / 64; ++it) {
        const int idx = it * 64 + lane;
        const int r = idx / CPRW, c = idx % CPRW;
        const int row = rbase + r, col = cur.n0 + wn * WN + c * 8;
        const u32x4 v = ld16(st_area + r * WN + ((c ^ (r % CPRW)) << 3));
        if (row < cur.m_end && col < p.N) {
          // weight gradients are written once and not read again by this pass: nontemporal
          // stores (32 experts of 256 rows, d = 7168, F = 2048: dW13 1308 -> 1188 us)
          if constexpr (MODE == BWD_KSEG)
            __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(yg + (int64_t)row * p.ldy + col));
          else
            st16(yg + (int64_t)row * p.ldy + col, v);
        }
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      __builtin_amdgcn_wave_barrier();
    }
    if (!more) break;
  }
}

template <int BM, int BN, int BK, int STAGES, int WGM, int WGN, bool XMN, bool WMN, int MODE, int OCC = 1,
          bool KTAIL = true>
hipError_t launch_bwd(const GemmBwdProblem& p, hipStream_t stream) {
  static OccCache occ;
  if (!KTAIL && p.K % BK) return hipErrorInvalidValue;
  const void* fn = reinterpret_cast<const void*>(&k_gemm_bwd<BM, BN, BK, STAGES, WGM, WGN, XMN, WMN, MODE, OCC, KTAIL>);
  const size_t lds = (size_t)STAGES * (BM + BN) * BK * sizeof(bf16_t);
  const size_t lds_static = (MODE == BWD_ROWS ? 3 : 2) * (kMaxGroups + 1) * sizeof(int) + 64;
  if (lds + lds_static > (size_t)lds_limit()) return hipErrorInvalidConfiguration;
  hipError_t err;
  const int per_cu = kernel_occupancy(occ, fn, 64 * WGM * WGN, lds, err);
  if (err != hipSuccess) return err;
  const int64_t tn = (p.N + BN - 1) / BN;
  const int64_t upper = MODE == BWD_ROWS ? tn * ((p.max_rows + BM - 1) / BM + p.groups)
                                         : (int64_t)p.groups * ((p.M + BM - 1) / BM) * tn;
  const int64_t resident = (int64_t)cu_count() * per_cu;
  int64_t grid = upper < resident ? upper : resident;
  if (grid >= 8) grid -= grid % 8;
  if (grid < 1) grid = 1;
  GemmBwdProblem arg = p;
  void* args[] = {&arg};
  hipError_t e = hipLaunchKernel(fn, dim3((unsigned)grid), dim3(64 * WGM * WGN), args, lds, stream);
  return e != hipSuccess ? e : hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_bwd(const GemmBwdProblem& p, hipStream_t stream) {
  if (p.groups < 1 || p.groups > kMaxGroups || p.N < 8 || p.N % 8 || p.offsets == nullptr)
    return hipErrorInvalidValue;
  if (p.seg_stride > 0 && (int64_t)p.groups * p.seg_stride > p.max_rows) return hipErrorInvalidValue;
  if (p.mode == BWD_ROWS) {
    // dA / dX: K-major activation rows against an MN-major weight
    if (p.x_mn || !p.w_mn || p.K < 8 || p.K % 8) return hipErrorInvalidValue;
    // K a multiple of 64 (every expert and shared dimension of the measured workloads): the
    // instances without K-tail code, which also leave the registers the 320-row tile needs
    const bool kt = p.K % 64 != 0;
    if (p.rows_hint > 0 && p.rows_hint <= 128)
      return kt ? launch_bwd<64, 128, 64, 3, 2, 2, false, true, BWD_ROWS, 1, true>(p, stream)
                : launch_bwd<64, 128, 64, 3, 2, 2, false, true, BWD_ROWS, 1, false>(p, stream);
    // Tile shapes (all on the MN-major weight operand, two ds_read_b64_tr_b16 per fragment):
    // 256 x 256 over 2 x 4 waves, a wave holding 128 token rows x 64 weight columns, so a K-step
    // reads four token fragments (ds_read_b128) and two weight fragments, against two and four
    // with 4 x 2 waves -- the transpose reads are the dearer ones (DeepSeek-V3 routed dX 816 ->
    // 634 us, shared dX 605 -> 481); 256 x 128 (4 x 2 waves); 320 x 256 (2 x 4 waves, 10 token
    // blocks).  Chosen like the forward's tiles, from the expected tile count of each shape: a
    // persistent launch takes about ceil(tiles / CUs) rounds, a 256 x 128 tile costs ~0.6 of a
    // 256 x 256 one and a 320-row tile ~1.15, and an expert's rows scatter around their mean with a
    // standard deviation of about its square root (at 256 rows per expert: 1.5 256-row m-tiles on
    // average, one 320-row tile).
    const double cus = cu_count();
    const double mu = p.rows_hint > 0 ? (double)p.rows_hint : (double)p.max_rows / p.groups;
    const double sigma = p.groups > 1 ? std::sqrt(mu) : 0.0;
    auto mtiles = [&](int bm) {
      double per_group = 0;
      if (sigma == 0) {
        per_group = std::ceil(mu / bm);
      } else {
        const int jmax = (int)((mu + 8 * sigma) / bm) + 1;
        for (int j = 0; j <= jmax; ++j)                   // E[ceil(m / bm)] = sum_j P(m > j bm)
          per_group += 0.5 * std::erfc((j * bm - mu) / (sigma * std::sqrt(2.0)));
      }
      return per_group * p.groups;
    };
    // rounds of the persistent grid; an expected count a few hundredths of a round above a
    // whole number (the normal tail of the row counts) is that whole number
    auto rounds = [&](double tiles) { return std::max(1.0, std::ceil(tiles / cus - 0.05)); };
    const double tn256 = (double)((p.N + 255) / 256), tn128 = (double)((p.N + 127) / 128);
    const double c1 = rounds(mtiles(256) * tn256), c2 = 0.6 * rounds(mtiles(256) * tn128);
    const double c3 = kt ? 1e30 : 1.15 * rounds(mtiles(320) * tn256);   // no tail instance of it
    int cfg = (c3 < c1 && c3 <= c2) ? 3 : c2 < c1 ? 2 : 1;
#ifdef MOE_BWD_ROWS_CFG
    cfg = MOE_BWD_ROWS_CFG;
#endif
    if (cfg == 3 && !kt) return launch_bwd<320, 256, 64, 2, 2, 4, false, true, BWD_ROWS, 1, false>(p, stream);
    if (cfg == 2)
      return kt ? launch_bwd<256, 128, 64, 3, 4, 2, false, true, BWD_ROWS, 1, true>(p, stream)
                : launch_bwd<256, 128, 64, 3, 4, 2, false, true, BWD_ROWS, 1, false>(p, stream);
    return kt ? launch_bwd<256, 256, 64, 2, 2, 4, false, true, BWD_ROWS, 1, true>(p, stream)
              : launch_bwd<256, 256, 64, 2, 2, 4, false, true, BWD_ROWS, 1, false>(p, stream);
  }
  if (p.mode == BWD_KSEG) {
    // weight gradients: both operands row-major activations reduced over the group's rows
    if (!p.x_mn || !p.w_mn || p.M < 8 || p.M % 8) return hipErrorInvalidValue;
    // 256 x 256 tiles, two 64-wide slices in flight: measured against 128 x 128 tiles with two
    // or three workgroups per CU and three 32-wide slices in flight (routed dW13 at DeepSeek-V3
    // 1079-1132 us against 985)
    // the router's weight gradient (float32 K-split partials, M = the expert count): 128 x 128
    // tiles, two workgroups per CU, 4x the tiles of 256 x 256 ones for its few output tiles
    // (DeepSeek-V3: 256 x 7168 outputs over 9 token chunks, 76 -> 59 us)
    if (p.Yf) return launch_bwd<128, 128, 64, 2, 2, 2, true, true, BWD_KSEG, 2>(p, stream);
#ifdef MOE_BWD_KSEG_CFG
    // tuning alternatives (not chosen by the launcher)
    switch (MOE_BWD_KSEG_CFG) {
      case 1: return launch_bwd<128, 128, 64, 2, 2, 2, true, true, BWD_KSEG, 2>(p, stream);
      case 3: return launch_bwd<128, 128, 32, 4, 2, 2, true, true, BWD_KSEG, 2>(p, stream);
      case 4: return launch_bwd<128, 128, 32, 3, 2, 2, true, true, BWD_KSEG, 3>(p, stream);
      default: break;
    }
#endif
    return launch_bwd<256, 256, 64, 2, 4, 2, true, true, BWD_KSEG, 1>(p, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace moe
