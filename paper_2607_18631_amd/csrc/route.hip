// Gating and top-k: one wavefront per token.
//
// The router logits come from the grouped GEMM (one group, float32 epilogue), possibly as
// nsplit partial sums over K chunks; they are added here in chunk order.  Lane l of the wave
// owns the PL contiguous experts [PL l, PL l + PL).  Every decision is taken on the float32
// key (softmax: logit + bias; sigmoid: the score): the larger key wins, equal keys go to the
// lower expert index, so the result does not depend on lane scheduling.
//
// Top-k, one expert per round: every key is mapped to a 32-bit unsigned integer with the same
// order (chosen and ineligible experts map to 0, below every key), the wave maximum of the lanes'
// largest values is taken with DPP moves (no LDS traffic), and of the lanes holding it the lowest
// lane wins (a ballot), inside it the lowest expert: equal keys go to the lower expert index.
//
// Group limit (n_group > 1): a group's score is the float32 sum of its two largest keys, and the
// topk_group groups with the largest scores stay eligible (equal scores: lower group index first).
// When each group is a run of 2, 4, 8 or 16 lanes, the scores come from DPP exchanges inside the
// run and every lane ranks its own group against the others' scores read from their lanes;
// otherwise the keys go through LDS, lane g scores and ranks group g, and a ballot of the ranks
// below topk_group is the mask of eligible groups.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace moe {
namespace {

constexpr int kMaxPerLane = 16;   // E <= 1024
constexpr int kWaves = 4;         // tokens per workgroup

// float -> uint32 with the same order (finite values and infinities; -0 counts as +0)
__device__ __forceinline__ uint32_t ordered(float f) {
  const uint32_t u = __float_as_uint(f + 0.0f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// the float key back from its ordered image (inverse of ordered)
__device__ __forceinline__ float unordered(uint32_t o) {
  return __uint_as_float((o & 0x80000000u) ? (o & 0x7fffffffu) : ~o);
}

// lanes of the rows in ROWS take src from the DPP pattern CTRL, the others 0 (the identity of an
// unsigned maximum, so each step below is one v_max_u32 with a DPP operand)
template <int CTRL, int ROWS = 0xf>
__device__ __forceinline__ uint32_t dppu(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROWS, 0xf, false);
}

// maximum over the 64 lanes, returned to every lane (wave-uniform)
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  v = max(v, dppu<0xb1>(v));              // quad_perm [1,0,3,2]
  v = max(v, dppu<0x4e>(v));              // quad_perm [2,3,0,1]
  v = max(v, dppu<0x141>(v));             // row_half_mirror: quads 0 <-> 1 of each 8
  v = max(v, dppu<0x140>(v));             // row_mirror: halves of each 16-lane row
  v = max(v, dppu<0x142, 0xa>(v));        // row_bcast:15 -> rows 1, 3 hold rows (0,1), (2,3)
  v = max(v, dppu<0x143, 0xc>(v));        // row_bcast:31 -> row 3 holds all four
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

template <int CTRL>
__device__ __forceinline__ float dppf(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), CTRL, 0xf, 0xf, false));
}

// merge the two-largest multisets (v1 >= v2) of this lane and the DPP partner lane
template <int CTRL>
__device__ __forceinline__ void top2_merge(float& v1, float& v2) {
  const float o1 = dppf<CTRL>(v1), o2 = dppf<CTRL>(v2);
  v2 = fmaxf(fminf(v1, o1), fmaxf(v2, o2));
  v1 = fmaxf(v1, o1);
}
// fixed-order sum / max over the 64 lanes (wave-uniform result)
__device__ __forceinline__ float wave_sum_fixed(float v) {
  v += dppf<0xb1>(v);
  v += dppf<0x4e>(v);
  v += dppf<0x141>(v);
  v += dppf<0x140>(v);
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return (r0 + r1) + (r2 + r3);
}
__device__ __forceinline__ float wave_max_fixed(float v) {
  v = fmaxf(v, dppf<0xb1>(v));
  v = fmaxf(v, dppf<0x4e>(v));
  v = fmaxf(v, dppf<0x141>(v));
  v = fmaxf(v, dppf<0x140>(v));
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return fmaxf(fmaxf(r0, r1), fmaxf(r2, r3));
}

template <int PL>
__global__ __launch_bounds__(64 * kWaves) void k_gate(GateProblem p) {
  __shared__ float s_key[kWaves][64 * PL];
  __shared__ float s_gscore[kWaves][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t t = (int64_t)blockIdx.x * kWaves + w;
  if (t >= p.T) return;                                   // wave-uniform
  const int E = p.E;
  const float NEG = -INFINITY;
  const int e0 = lane * PL;

  // ---- logits (sum of the K-chunk partials, chunk order) and keys ----
  // this lane's PL logits of one partial (16-byte loads where rows allow)
  auto load_row = [&](const float* row, float (&v)[PL]) {
    if constexpr (PL % 4 == 0) {
      if (E % 4 == 0) {
#pragma unroll
        for (int c = 0; c < PL / 4; ++c) {
          f32x4 q = {0.f, 0.f, 0.f, 0.f};
          if (e0 + 4 * c < E) q = *reinterpret_cast<const f32x4*>(row + e0 + 4 * c);
#pragma unroll
          for (int u = 0; u < 4; ++u) v[4 * c + u] = q[u];
        }
        return;
      }
    }
#pragma unroll
    for (int j = 0; j < PL; ++j) v[j] = (e0 + j < E) ? row[e0 + j] : 0.f;
  };
  float key[PL];
#pragma unroll
  for (int j = 0; j < PL; ++j) key[j] = 0.f;
  const float* row0 = p.logits + t * E;
  int s = 0;
  // NB partials' loads in flight (NB * PL <= 64 registers), added in chunk order
  constexpr int NB = PL <= 4 ? 8 : 64 / PL;
  for (; s + NB <= p.nsplit; s += NB) {
    float v[NB][PL];
#pragma unroll
    for (int u = 0; u < NB; ++u) load_row(row0 + (s + u) * p.split_stride, v[u]);
#pragma unroll
    for (int u = 0; u < NB; ++u)
#pragma unroll
      for (int j = 0; j < PL; ++j) key[j] += v[u][j];
  }
  if (s + NB / 2 <= p.nsplit) {
    float v[NB / 2][PL];
#pragma unroll
    for (int u = 0; u < NB / 2; ++u) load_row(row0 + (s + u) * p.split_stride, v[u]);
#pragma unroll
    for (int u = 0; u < NB / 2; ++u)
#pragma unroll
      for (int j = 0; j < PL; ++j) key[j] += v[u][j];
    s += NB / 2;
  }
  for (; s < p.nsplit; ++s) {
    float v[PL];
    load_row(row0 + s * p.split_stride, v);
#pragma unroll
    for (int j = 0; j < PL; ++j) key[j] += v[j];
  }
#pragma unroll
  for (int j = 0; j < PL; ++j) {
    const int e = e0 + j;
    float k = NEG;
    if (e < E) {
      const float L = key[j];
      k = (p.gate == 0) ? (p.bias ? L + p.bias[e] : L) : 1.0f / (1.0f + expf(-L));
      if (p.keys_out) p.keys_out[t * E + e] = k;
    }
    key[j] = k;
  }

  // ---- group limit ----
  uint32_t elig = 0;                                      // bit j: expert e0 + j may be chosen
#pragma unroll
  for (int j = 0; j < PL; ++j)
    if (e0 + j < E) elig |= 1u << j;
  if (p.n_group > 1) {
    const int ng = p.n_group, gsz = p.group_size;
    const int lpg = gsz / PL;                             // lanes per group when groups tile lanes
    if (gsz % PL == 0 && (lpg == 2 || lpg == 4 || lpg == 8 || lpg == 16)) {
      // each group is a run of lpg lanes inside one 16-lane row: the two largest keys by DPP
      // exchanges, after which every lane of the group holds the group's score
      float v1 = NEG, v2 = NEG;
#pragma unroll
      for (int j = 0; j < PL; ++j) {
        const float k = key[j];
        v2 = fmaxf(v2, fminf(v1, k));
        v1 = fmaxf(v1, k);
      }
      top2_merge<0xb1>(v1, v2);                           // pairs
      if (lpg >= 4) top2_merge<0x4e>(v1, v2);             // quads
      if (lpg >= 8) top2_merge<0x141>(v1, v2);            // 8 lanes
      if (lpg >= 16) top2_merge<0x140>(v1, v2);           // 16 lanes
      const float gs = v1 + v2;
      const int sh = __builtin_ctz((unsigned)lpg);
      const int g = lane >> sh;                           // this lane's group
      int rank = 0;                                       // groups ahead of it
      for (int h = 0; h < ng; ++h) {
        const float o = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(gs), h << sh));
        rank += (o > gs || (o == gs && h < g)) ? 1 : 0;
      }
      if (rank >= p.topk_group) elig = 0;
    } else {
      float gs = NEG;
#pragma unroll
      for (int j = 0; j < PL; ++j) s_key[w][e0 + j] = key[j];
      __builtin_amdgcn_wave_barrier();
      if (lane < ng) {
        float v1 = NEG, v2 = NEG;                         // two largest keys of the group
#pragma unroll 8
        for (int e = lane * gsz; e < (lane + 1) * gsz; ++e) {
          const float k = s_key[w][e];
          v2 = fmaxf(v2, fminf(v1, k));
          v1 = fmaxf(v1, k);
        }
        gs = v1 + v2;
        s_gscore[w][lane] = gs;
      }
      __builtin_amdgcn_wave_barrier();
      int rank = 0;
      if (lane < ng)
#pragma unroll 8
        for (int h = 0; h < ng; ++h) {
          const float o = s_gscore[w][h];
          rank += (o > gs || (o == gs && h < lane)) ? 1 : 0;
        }
      const uint64_t keep = __ballot(lane < ng && rank < p.topk_group);
      int g = e0 / gsz, r = e0 - g * gsz;                 // group of expert e0 + j, walked along j
#pragma unroll
      for (int j = 0; j < PL; ++j) {
        if (e0 + j < E && !((keep >> g) & 1ull)) elig &= ~(1u << j);
        if (++r == gsz) {
          r = 0;
          ++g;
        }
      }
    }
  }

  // ---- top-k: k rounds of wave argmax over eligible, not yet chosen keys ----
  uint32_t uk[PL];                                        // ordered keys; 0: not selectable
#pragma unroll
  for (int j = 0; j < PL; ++j) uk[j] = ((elig >> j) & 1u) ? ordered(key[j]) : 0u;
  float selk[16];
  int seli[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    selk[r] = 0.f;
    seli[r] = 0;
    if (r < p.top_k) {
      uint32_t best = uk[0];
#pragma unroll
      for (int j = 1; j < PL; ++j) best = max(best, uk[j]);
      const uint32_t m = wave_max_u32(best);
      // lowest lane holding the maximum (some lane does), then its lowest expert holding it
      const int wl = __builtin_ctzll(__ballot(best == m));
      int jf = PL - 1;
#pragma unroll
      for (int j = PL - 2; j >= 0; --j) jf = (uk[j] == m) ? j : jf;
      const int jw = __builtin_amdgcn_readlane(jf, wl);
      // (the host guarantees at least top_k eligible experts, so m names one)
      seli[r] = min(wl * PL + jw, E - 1);
      selk[r] = unordered(m);
#pragma unroll
      for (int j = 0; j < PL; ++j) uk[j] = (lane == wl && j == jw) ? 0u : uk[j];
    }
  }

  // ---- gates (float32, slot order) ----
  float den = 0.f;
  float m = selk[0];
  if (p.gate == 0 && !p.renormalize) {
    float mm = NEG;
#pragma unroll
    for (int j = 0; j < PL; ++j) mm = fmaxf(mm, key[j]);
    m = wave_max_fixed(mm);
    float part = 0.f;
#pragma unroll
    for (int j = 0; j < PL; ++j)
      if (e0 + j < E) part += expf(key[j] - m);
    den = wave_sum_fixed(part);
  }
  float wgt[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    wgt[r] = 0.f;
    if (r < p.top_k) {
      wgt[r] = (p.gate == 0) ? expf(selk[r] - m) : selk[r];
      if (p.renormalize) den += wgt[r];
    }
  }
  const bool divide = p.renormalize || p.gate == 0;
  // lane r < top_k writes slot r
  int oi = 0;
  float ow = 0.f;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    if (r < p.top_k) {
      oi = (lane == r) ? seli[r] : oi;
      ow = (lane == r) ? wgt[r] : ow;
    }
  }
  ow = (divide ? ow / den : ow) * p.routed_scale;
  if (lane < p.top_k) {
    p.topk_idx[t * p.top_k + lane] = oi;
    p.topk_w[t * p.top_k + lane] = ow;
  }
}

template <int PL>
hipError_t launch_pl(const GateProblem& p, hipStream_t stream) {
  const unsigned blocks = (unsigned)((p.T + kWaves - 1) / kWaves);
  hipLaunchKernelGGL(k_gate<PL>, dim3(blocks), dim3(64 * kWaves), 0, stream, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gate(const GateProblem& p, hipStream_t stream) {
  if (p.nsplit < 1) return hipErrorInvalidValue;
  const int pl = (p.E + 63) / 64;
  if (pl <= 1) return launch_pl<1>(p, stream);
  if (pl <= 2) return launch_pl<2>(p, stream);
  if (pl <= 4) return launch_pl<4>(p, stream);
  if (pl <= 8) return launch_pl<8>(p, stream);
  if (pl <= kMaxPerLane) return launch_pl<16>(p, stream);
  return hipErrorInvalidValue;
}

}  // namespace moe
