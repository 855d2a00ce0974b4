// Gating and top-k: one wavefront per token.
//
// The router logits come from the grouped GEMM (one group, float32 epilogue).  Lane l of
// the wave owns experts l, l + 64, l + 128, ... (up to 16 per lane for E <= 1024).  Every
// decision is taken on the float32 key (softmax: logit + bias; sigmoid: the score), with
// wave-wide butterfly argmax reductions: the larger key wins, equal keys go to the lower
// expert index, so the result does not depend on lane scheduling.
//
// Group limit (n_group > 1): each contiguous group scores the float32 sum of its two
// largest keys (two argmax passes per group), the topk_group best groups stay eligible.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace moe {
namespace {

constexpr int kMaxPerLane = 16;   // E <= 1024

template <int PL>
__global__ __launch_bounds__(256) void k_gate(GateProblem p) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= p.T) return;
  const int E = p.E;
  const float NEG = -INFINITY;

  float key[PL];
  const float* lrow = p.logits + t * E;
#pragma unroll
  for (int i = 0; i < PL; ++i) {
    const int e = i * 64 + lane;
    float k = NEG;
    if (e < E) {
      const float L = lrow[e];
      if (p.gate == 0) {
        k = p.bias ? L + p.bias[e] : L;
      } else {
        k = 1.0f / (1.0f + expf(-L));
      }
      if (p.keys_out) p.keys_out[t * E + e] = k;
    }
    key[i] = k;
  }

  // ---- group limit: lane g holds the score of group g ----
  bool elig[PL];
#pragma unroll
  for (int i = 0; i < PL; ++i) elig[i] = (i * 64 + lane) < E;
  if (p.n_group > 1) {
    const int gsz = E / p.n_group;
    float my_gscore = NEG;
    for (int g = 0; g < p.n_group; ++g) {
      const int lo = g * gsz, hi = lo + gsz;
      float v1 = NEG;
      int i1 = 0x7fffffff;
#pragma unroll
      for (int i = 0; i < PL; ++i) {
        const int e = i * 64 + lane;
        if (e >= lo && e < hi && (key[i] > v1 || (key[i] == v1 && e < i1))) { v1 = key[i]; i1 = e; }
      }
      wave_argmax(v1, i1);
      float v2 = NEG;
      int i2 = 0x7fffffff;
#pragma unroll
      for (int i = 0; i < PL; ++i) {
        const int e = i * 64 + lane;
        if (e >= lo && e < hi && e != i1 && (key[i] > v2 || (key[i] == v2 && e < i2))) { v2 = key[i]; i2 = e; }
      }
      wave_argmax(v2, i2);
      if (lane == g) my_gscore = v1 + v2;
    }
    uint64_t keep = 0;
    for (int s = 0; s < p.topk_group; ++s) {
      float v = ((keep >> lane) & 1ull) ? NEG : my_gscore;
      int gi = (lane < p.n_group && !((keep >> lane) & 1ull)) ? lane : 0x7fffffff;
      wave_argmax(v, gi);
      keep |= 1ull << gi;
    }
#pragma unroll
    for (int i = 0; i < PL; ++i) {
      const int e = i * 64 + lane;
      elig[i] = elig[i] && e < E && ((keep >> (min(e / gsz, 63))) & 1ull);
    }
  }

  // ---- top-k: k rounds of wave argmax over eligible, not yet chosen keys ----
  float selk[16];
  int seli[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    selk[j] = 0.f;
    seli[j] = 0;
    if (j < p.top_k) {
      float v = NEG;
      int idx = 0x7fffffff;
#pragma unroll
      for (int i = 0; i < PL; ++i) {
        const int e = i * 64 + lane;
        if (elig[i] && (idx == 0x7fffffff || key[i] > v || (key[i] == v && e < idx))) { v = key[i]; idx = e; }
      }
      wave_argmax(v, idx);
      selk[j] = v;
      seli[j] = idx;
#pragma unroll
      for (int i = 0; i < PL; ++i)
        if (i * 64 + lane == idx) elig[i] = false;
    }
  }

  // ---- gates (float32, slot order) ----
  float den = 0.f;
  float m = selk[0];
  if (p.gate == 0 && !p.renormalize) {
    float mm = NEG;
#pragma unroll
    for (int i = 0; i < PL; ++i) mm = fmaxf(mm, key[i]);
    m = wave_max(mm);
    float part = 0.f;
#pragma unroll
    for (int i = 0; i < PL; ++i)
      if (i * 64 + lane < E) part += expf(key[i] - m);
    den = wave_sum(part);
  }
  float w[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    w[j] = 0.f;
    if (j < p.top_k) {
      w[j] = (p.gate == 0) ? expf(selk[j] - m) : selk[j];
      if (p.renormalize) den += w[j];
    }
  }
  const bool divide = p.renormalize || p.gate == 0;
  int oi = 0;
  float ow = 0.f;
#pragma unroll
  for (int j = 0; j < 16; ++j)
    if (j == lane) { oi = seli[j]; ow = (divide ? w[j] / den : w[j]) * p.routed_scale; }
  if (lane < p.top_k) {
    p.topk_idx[t * p.top_k + lane] = oi;
    p.topk_w[t * p.top_k + lane] = ow;
  }
}

template <int PL>
hipError_t launch_pl(const GateProblem& p, hipStream_t stream) {
  const unsigned blocks = (unsigned)((p.T + 3) / 4);
  hipLaunchKernelGGL(k_gate<PL>, dim3(blocks), dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gate(const GateProblem& p, hipStream_t stream) {
  const int pl = (p.E + 63) / 64;
  if (pl <= 1) return launch_pl<1>(p, stream);
  if (pl <= 2) return launch_pl<2>(p, stream);
  if (pl <= 4) return launch_pl<4>(p, stream);
  if (pl <= 8) return launch_pl<8>(p, stream);
  if (pl <= kMaxPerLane) return launch_pl<16>(p, stream);
  return hipErrorInvalidValue;
}

}  // namespace moe
