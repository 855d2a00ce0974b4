// Histogram, prefix scan and stable permutation of the local (token, expert) slots.
//
// Tokens are cut into super-chunks of 512 (eight 64-token chunks, one wavefront each).  Two
// launches (three for very wide count tables):
//   k_super_rank  per super-chunk (one wave per chunk): for every chunk and local expert, the
//                 64-bit mask of the chunk's lanes (tokens) holding that expert and the chunk's
//                 base inside the super-chunk (a scan of the eight chunks' counts), and the
//                 super-chunk's count per local expert
//   k_super_scan  (only when the super-chunk x expert count table is large) per expert, the
//                 exclusive scan of the counts over super-chunks and the expert total
//   k_place_*     per token: the expert bases of its super-chunk and the offsets (exclusive
//                 scan of the expert totals, the monotone [E_local+1] array) from the count
//                 table, each slot's rank (its chunk's base plus the popcount of its expert's
//                 mask below its lane), hence its row
//                     row = offsets[e] + base[super-chunk][e] + rank,
//                 then slot_row / row_token (and the gate of each row when asked), counts and
//                 offsets (first workgroup), and -- in the copy forms, one wavefront per token --
//                 the bit-exact copy of the token row to each of its local rows.  The copy forms
//                 issue the token row's loads before they read the tables, so the tables'
//                 latency hides behind them.
//
// Masked-decode layout (expert capacity C > 0): expert e's rows are e * C + rank for the
// ranks below C; later slots are dropped (slot_row = -1) and offsets[e] = e * C.
//
// The ranks need no ordering of atomics: each chunk's lane masks are the same whatever order
// the LDS ORs land in, so the order inside an expert is ascending token (a stable counting
// sort) and run-to-run identical.  Two slots of one token never share an expert, so a token
// sets at most one bit of a mask.
#include <mutex>

#include "common.hpp"
#include "kernels.hpp"

namespace moe {
namespace {

constexpr int CH = kPermChunk;   // tokens per chunk = lanes of one wave
constexpr int SCW = kPermSuper;  // chunks (waves) per super-chunk
constexpr int SC = CH * SCW;     // tokens per super-chunk
// count tables of at most this many super-chunks and entries (super-chunks x local experts) are
// scanned by every k_place workgroup itself; larger ones by k_super_scan first
constexpr int64_t kInlineSupers = 64;
constexpr int64_t kInlineTable = 4096;

// one wave per chunk: for every local expert the 64-bit mask of the chunk's lanes (tokens) with a
// slot of that expert, built with LDS atomic ORs (order-independent, so deterministic); a slot's
// rank inside the chunk is the popcount of its expert's mask below its lane and the chunk's count
// of an expert the popcount of the whole mask
__global__ __launch_bounds__(64 * SCW) void k_super_rank(PermuteProblem p) {
  extern __shared__ uint64_t s_mask[];         // [SCW][E_local] lane masks, then [SCW][E_local] int bases
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int s = blockIdx.x;
  const int E_local = p.E_local, k = p.top_k;
  int* s_base = reinterpret_cast<int*>(s_mask + SCW * E_local);
  for (int i = tid; i < SCW * E_local; i += 64 * SCW) s_mask[i] = 0ull;
  const int64_t t = (int64_t)s * SC + w * CH + lane;
  const bool valid_t = t < p.T;
  int myle[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    myle[j] = -1;
    if (j < k && valid_t) {
      const int le = p.topk_idx[t * k + j] - p.e_begin;
      myle[j] = (le >= 0 && le < E_local) ? le : -1;
    }
  }
  __syncthreads();
  uint64_t* mask = s_mask + w * E_local;
#pragma unroll
  for (int j = 0; j < 16; ++j)
    if (j < k && myle[j] >= 0) atomicOr(reinterpret_cast<unsigned long long*>(&mask[myle[j]]), 1ull << lane);
  __syncthreads();
  // per expert: the chunks' bases inside the super-chunk (exclusive scan of the chunk counts) and
  // the super-chunk's total
  for (int e = tid; e < E_local; e += 64 * SCW) {
    int run = 0;
#pragma unroll
    for (int c = 0; c < SCW; ++c) {
      s_base[c * E_local + e] = run;
      run += __popcll(s_mask[c * E_local + e]);
    }
    p.super_count[(int64_t)s * E_local + e] = run;
  }
  __syncthreads();                             // every expert's bases written before they are stored
  // the chunks' masks and bases inside the super-chunk, for the placement launch
  for (int i = tid; i < SCW * E_local; i += 64 * SCW) {
    const int64_t at = (int64_t)s * SCW * E_local + i;        // chunk s * SCW + i / E_local, expert i % E_local
    p.chunk_mask[at] = s_mask[i];
    p.chunk_base[at] = s_base[i];
  }
}

// rank of token t's slot of local expert le among the earlier slots of le in t's super-chunk
__device__ __forceinline__ int slot_rank(const PermuteProblem& p, int64_t t, int le) {
  const int64_t at = (t / CH) * p.E_local + le;
  const int pos = (int)(t % CH);
  const uint64_t below = pos == 0 ? 0ull : (~0ull >> (64 - pos));
  return p.chunk_base[at] + (int)__popcll(p.chunk_mask[at] & below);
}

// one workgroup per local expert: exclusive scan of super_count[:, e] over super-chunks, and
// the expert total (wide count tables only)
__global__ __launch_bounds__(256) void k_super_scan(PermuteProblem p, int nsuper) {
  __shared__ int s_w[4];
  const int e = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int carry = 0;
  for (int b0 = 0; b0 < nsuper; b0 += 256) {
    const int b = b0 + tid;
    const int v = b < nsuper ? p.super_count[(int64_t)b * p.E_local + e] : 0;
    int inc = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int n = __shfl_up(inc, o, 64);
      if (lane >= o) inc += n;
    }
    if (lane == 63) s_w[wave] = inc;
    __syncthreads();
    int wbase = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      if (w < wave) wbase += s_w[w];
      tot += s_w[w];
    }
    if (b < nsuper) p.super_base[(int64_t)b * p.E_local + e] = carry + wbase + inc - v;
    carry += tot;
    __syncthreads();
  }
  if (tid == 0) p.totals[e] = carry;
}

// Expert bases of super-chunk s and the offsets, into LDS: s_base[e] = rows of expert e in the
// super-chunks before s, s_off[e] = exclusive scan of the expert totals (e * C in the masked
// layout), s_off[E_local] = their sum.  The first workgroup also writes counts and offsets.
// 256 threads: first one expert per thread (the super-chunk loop unrolled, so its loads are in
// flight together), then a scan of the totals with up to PER consecutive experts per thread.
__device__ void place_table(const PermuteProblem& p, int s, int nsuper, bool scanned, int* s_base, int* s_off,
                            int* s_tot, int* s_w) {
  constexpr int PER = 4;                       // 256 threads x 4 >= 1024 experts
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int E_local = p.E_local;
  for (int e = tid; e < E_local; e += 256) {
    int base = 0, tot = 0;
    if (scanned) {
      base = p.super_base[(int64_t)s * E_local + e];
      tot = p.totals[e];
    } else {
      const int32_t* col = p.super_count + e;
#pragma unroll 16
      for (int q = 0; q < nsuper; ++q) {
        const int v = col[(int64_t)q * E_local];
        base += q < s ? v : 0;
        tot += v;
      }
    }
    s_base[e] = base;
    s_tot[e] = tot;
  }
  __syncthreads();
  int tot[PER], lsum = 0;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int e = tid * PER + i;
    tot[i] = e < E_local ? s_tot[e] : 0;
    lsum += tot[i];
  }
  int inc = lsum;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int n = __shfl_up(inc, o, 64);
    if (lane >= o) inc += n;
  }
  if (lane == 63) s_w[wave] = inc;
  __syncthreads();
  int run = 0, all = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    if (w < wave) run += s_w[w];
    all += s_w[w];
  }
  run += inc - lsum;
  const int C = p.expert_capacity;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int e = tid * PER + i;
    if (e < E_local) {
      s_off[e] = C > 0 ? e * C : run;
      if (blockIdx.x == 0) {
        p.counts[e] = tot[i];
        p.offsets[e] = s_off[e];
      }
    }
    run += tot[i];
  }
  if (tid == 0) {
    s_off[E_local] = C > 0 ? E_local * C : all;
    if (blockIdx.x == 0) p.offsets[E_local] = s_off[E_local];
  }
  __syncthreads();
}

// row of a local slot from its expert and its rank inside its super-chunk (-1: dropped)
__device__ __forceinline__ int place_row(const PermuteProblem& p, const int* s_base, const int* s_off, int le,
                                         int srank) {
  if (le < 0 || srank < 0) return -1;
  const int grank = s_base[le] + srank;                  // rank inside the expert
  int row;
  if (p.expert_capacity > 0)                             // masked-decode layout: drop past C
    row = grank < p.expert_capacity ? le * p.expert_capacity + grank : -1;
  else
    row = s_off[le] + grank;
  return row < p.cap ? row : -1;        // unreachable for a consistent count table; keeps writes in bounds
}

// Copy form: one wave per token (PT tokens of one super-chunk per workgroup); the token row is
// read once (16-byte vectors, U per lane in flight, issued before the count table is read) and
// written to each of its local rows.
constexpr int PT = 4;
__global__ __launch_bounds__(64 * PT) void k_place_copy(PermuteProblem p, int nsuper, int scanned) {
  constexpr int U = 16;
  extern __shared__ int s_tab[];               // [E_local] bases, [E_local + 1] offsets, [E_local] totals
  __shared__ int s_w[4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int k = p.top_k, E_local = p.E_local;
  const int64_t t0 = (int64_t)blockIdx.x * PT;
  const int s = (int)(t0 / SC);
  const int64_t t = t0 + wave;
  const bool valid_t = t < p.T;
  int le[16], srank[16];
  bool any = false;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    le[j] = -1;
    srank[j] = -1;
    if (j < k && valid_t) {
      const int l = p.topk_idx[t * k + j] - p.e_begin;
      le[j] = (l >= 0 && l < E_local) ? l : -1;
      if (le[j] >= 0) srank[j] = slot_rank(p, t, l);
      any |= le[j] >= 0;
    }
  }
  const int nvec = p.d / 8;
  const u32x4* src = reinterpret_cast<const u32x4*>(p.x + (valid_t ? t : 0) * p.d);
  u32x4 val[U];
  if (any) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = u * 64 + lane;
      if (v < nvec) val[u] = src[v];
    }
  }
  place_table(p, s, nsuper, scanned != 0, s_tab, s_tab + E_local, s_tab + 2 * E_local + 1, s_w);
  if (!valid_t) return;
  int rows[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    rows[j] = (j < k) ? place_row(p, s_tab, s_tab + E_local, le[j], srank[j]) : -1;
    if (j < k && lane == j) {
      p.slot_row[t * k + j] = rows[j];
      if (rows[j] >= 0) {
        p.row_token[rows[j]] = (int32_t)t;
        if (p.row_weight) p.row_weight[rows[j]] = p.topk_w[t * k + j];
      }
    }
  }
  if (!any) return;
  for (int v0 = 0; v0 < nvec; v0 += 64 * U) {
    if (v0 > 0) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int v = v0 + u * 64 + lane;
        if (v < nvec) val[u] = src[v];
      }
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if (rows[j] < 0) continue;
      u32x4* dst = reinterpret_cast<u32x4*>(p.x_perm + (int64_t)rows[j] * p.d);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int v = v0 + u * 64 + lane;
        if (v < nvec) dst[v] = val[u];
      }
    }
  }
}

// The expert table of super-chunk s held by one wave (up to 64 local experts, at most
// kInlineSupers super-chunks): lane l ends with pre = rows of expert l % EP in the super-chunks
// before s and off = its offset (e * C in the masked layout).  Lane l first sums the super-chunks
// q = g, g + NG, ... of expert e = l % EP, g = l / EP (EP = E_local rounded up to a power of two,
// NG = 64 / EP lane groups); the groups' sums are combined by xor-shuffles and the totals scanned
// within EP lanes.  `first` writes counts and offsets.
// wave_table in two parts: the lane's sums over its super-chunks (issued first, as they depend on
// nothing else), then the shuffles
__device__ __forceinline__ void wave_table_sums(const PermuteProblem& p, int s, int nsuper, int ep, int& pre,
                                                int& tot) {
  const int lane = threadIdx.x & 63, E_local = p.E_local;
  const int e = lane & (ep - 1), g = lane / ep, ng = 64 / ep;
  tot = 0;
  pre = 0;
  if (e < E_local) {
#pragma unroll 8
    for (int q = g; q < nsuper; q += ng) {
      const int v = p.super_count[(int64_t)q * E_local + e];
      pre += q < s ? v : 0;
      tot += v;
    }
  }
}
__device__ __forceinline__ void wave_table_finish(const PermuteProblem& p, int ep, bool first, int& pre, int tot,
                                                  int& off) {
  const int lane = threadIdx.x & 63, E_local = p.E_local;
  const int e = lane & (ep - 1);
  for (int o = ep; o < 64; o <<= 1) {
    pre += __shfl_xor(pre, o, 64);
    tot += __shfl_xor(tot, o, 64);
  }
  int inc = tot;                                // inclusive scan of the totals over e (EP lanes)
  for (int o = 1; o < ep; o <<= 1) {
    const int n = __shfl_up(inc, o, 64);
    if (e >= o) inc += n;
  }
  const int C = p.expert_capacity;
  off = C > 0 ? e * C : inc - tot;
  if (first && lane < E_local) {
    p.counts[lane] = tot;
    p.offsets[lane] = off;
    if (lane == E_local - 1) p.offsets[E_local] = C > 0 ? E_local * C : inc;
  }
}
__device__ __forceinline__ void wave_table(const PermuteProblem& p, int s, int nsuper, int ep, bool first, int& pre,
                                           int& off) {
  int tot;
  wave_table_sums(p, s, nsuper, ep, pre, tot);
  wave_table_finish(p, ep, first, pre, tot, off);
}

// Copy form for up to 64 local experts and a count table of at most kInlineSupers super-chunks:
// one wave per workgroup and token, the expert bases and offsets computed by the wave itself
// with lane shuffles (no LDS, no barrier), so the table's latency of one wave overlaps the row
// traffic of the others on its compute unit.
__global__ __launch_bounds__(64) void k_place_wave(PermuteProblem p, int nsuper, int ep) {
  constexpr int U = 8;
  const int lane = threadIdx.x;
  const int k = p.top_k, E_local = p.E_local;
  const int64_t t = blockIdx.x;
  const int s = (int)(t / SC);
  int pre, tot, off;
  wave_table_sums(p, s, nsuper, ep, pre, tot);
  int le[16], srank[16];
  bool any = false;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    le[j] = -1;
    srank[j] = -1;
    if (j < k) {
      const int l = p.topk_idx[t * k + j] - p.e_begin;
      le[j] = (l >= 0 && l < E_local) ? l : -1;
      if (le[j] >= 0) srank[j] = slot_rank(p, t, l);
      any |= le[j] >= 0;
    }
  }
  const int nvec = p.d / 8;
  const u32x4* src = reinterpret_cast<const u32x4*>(p.x + t * p.d);
  u32x4 val[U];
  if (any) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = u * 64 + lane;
      if (v < nvec) val[u] = src[v];
    }
  }
  wave_table_finish(p, ep, t == 0, pre, tot, off);
  const int C = p.expert_capacity;
  int rows[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    rows[j] = -1;
    if (j < k) {
      const int l = le[j] < 0 ? 0 : le[j];
      const int base = __shfl(pre, l, 64), o = __shfl(off, l, 64);
      if (le[j] >= 0) {
        const int grank = base + srank[j];
        int row = C > 0 ? (grank < C ? le[j] * C + grank : -1) : o + grank;
        rows[j] = row < p.cap ? row : -1;
      }
      if (lane == j) {
        p.slot_row[t * k + j] = rows[j];
        if (rows[j] >= 0) {
          p.row_token[rows[j]] = (int32_t)t;
          if (p.row_weight) p.row_weight[rows[j]] = p.topk_w[t * k + j];
        }
      }
    }
  }
  if (!any) return;
  for (int v0 = 0; v0 < nvec; v0 += 64 * U) {
    if (v0 > 0) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int v = v0 + u * 64 + lane;
        if (v < nvec) val[u] = src[v];
      }
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if (rows[j] < 0) continue;
      u32x4* dst = reinterpret_cast<u32x4*>(p.x_perm + (int64_t)rows[j] * p.d);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int v = v0 + u * 64 + lane;
        if (v < nvec) __builtin_nontemporal_store(val[u], dst + v);   // streamed, not kept in the caches
      }
    }
  }
}

// Index form for up to 64 local experts and at most kInlineSupers super-chunks: one wave per 64
// tokens (one lane each), the table held by the wave (wave_table), each lane reading its
// experts' entries with a per-lane shuffle.
__global__ __launch_bounds__(64) void k_place_index_wave(PermuteProblem p, int nsuper, int ep) {
  const int lane = threadIdx.x;
  const int k = p.top_k, E_local = p.E_local;
  const int64_t t = (int64_t)blockIdx.x * 64 + lane;
  const int s = (int)(((int64_t)blockIdx.x * 64) / SC);
  const bool valid_t = t < p.T;
  int le[16], srank[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    le[j] = -1;
    srank[j] = -1;
    if (j < k && valid_t) {
      const int l = p.topk_idx[t * k + j] - p.e_begin;
      le[j] = (l >= 0 && l < E_local) ? l : -1;
      if (le[j] >= 0) srank[j] = slot_rank(p, t, l);
    }
  }
  int pre, off;
  wave_table(p, s, nsuper, ep, blockIdx.x == 0, pre, off);
  const int C = p.expert_capacity;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    if (j < k) {
      const int l = le[j] < 0 ? 0 : le[j];
      const int base = __shfl(pre, l, 64), o = __shfl(off, l, 64);
      int row = -1;
      if (le[j] >= 0) {
        const int grank = base + srank[j];
        row = C > 0 ? (grank < C ? le[j] * C + grank : -1) : o + grank;
        if (row >= p.cap) row = -1;
      }
      if (valid_t) {
        p.slot_row[t * k + j] = row;
        if (row >= 0) {
          p.row_token[row] = (int32_t)t;
          if (p.row_weight) p.row_weight[row] = p.topk_w[t * k + j];
        }
      }
    }
  }
}

// Index form (no row copy: the caller's GEMM reads the token rows through row_token): one
// thread per token, PI tokens of one super-chunk per workgroup.
constexpr int PI = 256;
__global__ __launch_bounds__(PI) void k_place_index(PermuteProblem p, int nsuper, int scanned) {
  extern __shared__ int s_tab[];               // [E_local] bases, [E_local + 1] offsets, [E_local] totals
  __shared__ int s_w[4];
  const int k = p.top_k, E_local = p.E_local;
  const int64_t t0 = (int64_t)blockIdx.x * PI;
  const int s = (int)(t0 / SC);
  const int64_t t = t0 + threadIdx.x;
  const bool valid_t = t < p.T;
  int le[16], srank[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    le[j] = -1;
    srank[j] = -1;
    if (j < k && valid_t) {
      const int l = p.topk_idx[t * k + j] - p.e_begin;
      le[j] = (l >= 0 && l < E_local) ? l : -1;
      if (le[j] >= 0) srank[j] = slot_rank(p, t, l);
    }
  }
  place_table(p, s, nsuper, scanned != 0, s_tab, s_tab + E_local, s_tab + 2 * E_local + 1, s_w);
  if (!valid_t) return;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    if (j < k) {
      const int row = place_row(p, s_tab, s_tab + E_local, le[j], srank[j]);
      p.slot_row[t * k + j] = row;
      if (row >= 0) {
        p.row_token[row] = (int32_t)t;
        if (p.row_weight) p.row_weight[row] = p.topk_w[t * k + j];
      }
    }
  }
}

// one wave per token: the token row is read once (16-byte vectors, U per lane in flight)
// and written to each of its local rows
__global__ __launch_bounds__(256) void k_gather(PermuteProblem p) {
  constexpr int U = 8;
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= p.T) return;
  const int k = p.top_k;
  int rows[16];
  bool any = false;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    rows[j] = (j < k) ? p.slot_row[t * k + j] : -1;
    if (rows[j] >= p.cap) rows[j] = -1;
    any |= rows[j] >= 0;
  }
  if (!any) return;
  const int nvec = p.d / 8;
  const u32x4* src = reinterpret_cast<const u32x4*>(p.x + t * p.d);
  for (int v0 = 0; v0 < nvec; v0 += 64 * U) {
    u32x4 val[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = v0 + u * 64 + lane;
      if (v < nvec) val[u] = src[v];
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if (rows[j] < 0) continue;
      u32x4* dst = reinterpret_cast<u32x4*>(p.x_perm + (int64_t)rows[j] * p.d);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int v = v0 + u * 64 + lane;
        if (v < nvec) dst[v] = val[u];
      }
    }
  }
}

}  // namespace

namespace {
// k_super_rank's LDS (12 bytes per chunk and local expert) exceeds the default 64 KB dynamic limit
// for more than 682 local experts: its limit is raised to the largest request once per device
struct RankLds {
  std::once_flag once;
  hipError_t err = hipSuccess;
};
RankLds g_rank_lds[kMaxDevices];
constexpr size_t kRankLdsMax = SCW * kMaxGroups * (sizeof(uint64_t) + sizeof(int));
}  // namespace

hipError_t launch_permute(const PermuteProblem& p, hipStream_t stream, int (*between)()) {
  const int64_t nsuper = permute_supers(p.T);
  const size_t rank_lds = SCW * p.E_local * (sizeof(uint64_t) + sizeof(int));
  if (rank_lds > 65536) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    RankLds& r = g_rank_lds[dev];
    std::call_once(r.once, [&] {
      r.err = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_super_rank),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, (int)kRankLdsMax);
    });
    if (r.err != hipSuccess) return r.err;
  }
  hipLaunchKernelGGL(k_super_rank, dim3((unsigned)nsuper), dim3(64 * SCW), rank_lds, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const bool scanned = nsuper > kInlineSupers || nsuper * p.E_local > kInlineTable;
  if (scanned) {
    hipLaunchKernelGGL(k_super_scan, dim3((unsigned)p.E_local), dim3(256), 0, stream, p, (int)nsuper);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (between && between() != 0) return hipErrorUnknown;
  const size_t tab = (3 * (size_t)p.E_local + 1) * sizeof(int);
  int ep = 1;
  while (ep < p.E_local) ep <<= 1;
  const bool wave_tab = !scanned && p.E_local <= 64;
  if (p.x_perm == nullptr && wave_tab) {
    hipLaunchKernelGGL(k_place_index_wave, dim3((unsigned)((p.T + 63) / 64)), dim3(64), 0, stream, p, (int)nsuper, ep);
  } else if (p.x_perm == nullptr) {
    hipLaunchKernelGGL(k_place_index, dim3((unsigned)((p.T + PI - 1) / PI)), dim3(PI), tab, stream, p, (int)nsuper,
                       (int)scanned);
  } else if (wave_tab) {
    hipLaunchKernelGGL(k_place_wave, dim3((unsigned)p.T), dim3(64), 0, stream, p, (int)nsuper, ep);
  } else {
    hipLaunchKernelGGL(k_place_copy, dim3((unsigned)((p.T + PT - 1) / PT)), dim3(64 * PT), tab, stream, p,
                       (int)nsuper, (int)scanned);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// Library-owned scratch for moe_permute_noalloc: the per-chunk counts and bases live in a
// file-scope device array instead of a caller workspace.  Each device holds its own copy;
// host code never uses the array's name as an address (on the host it is only a symbol
// handle), it uses the address hipGetSymbolAddress returns on that device.
// ---------------------------------------------------------------------------------------
static __device__ __align__(256) uint8_t scratch[kPermuteScratchBytes];

namespace {
struct ScratchAddr {
  std::once_flag once;
  void* ptr = nullptr;
  hipError_t err = hipSuccess;
};
ScratchAddr g_scratch[kMaxDevices];
}  // namespace

hipError_t permute_scratch(void** ptr) {
  *ptr = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  ScratchAddr& s = g_scratch[dev];
  // once per device, with that device current (hipGetDevice above is the calling thread's)
  std::call_once(s.once, [&] { s.err = hipGetSymbolAddress(&s.ptr, HIP_SYMBOL(scratch)); });
  if (s.err != hipSuccess) return s.err;
  if (s.ptr == nullptr) return hipErrorInvalidSymbol;
  *ptr = s.ptr;
  return hipSuccess;
}

hipError_t launch_gather(const PermuteProblem& p, hipStream_t stream) {
  if (p.T <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_gather, dim3((unsigned)((p.T + 3) / 4)), dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace moe
