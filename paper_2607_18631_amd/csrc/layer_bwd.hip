// Kernels of the layer backward around the expert-MLP backward GEMMs: the combine's backward
// (gate gradients and the gradients of the expert output rows), the gating / router-logit
// backward, and the sum of every token's row gradients.  One wavefront per token in each, no
// atomics: every result is bit-identical from run to run.
//
// With out[t] = sum_j w_tj y_{t,j} + y_s[t] (the combine), for output gradient g = dout[t]:
//   dgate[t, j]          = <g, y_{t,j}>        (local slots; 0 for slots routed elsewhere)
//   dy_perm[row(t, j)]   = w_tj g              (the expert rows' output gradients)
// The gates are functions of the float32 keys the forward decided on (recomputed here from
// the same logit partials, in the same order), the choice of experts carries no gradient:
//   softmax, renormalised:  w_j = s p_j, p = softmax over the chosen keys
//                           dkey_j = s p_j (dgate_j - sum_i p_i dgate_i)
//   softmax over all E:     w_j = s P_j,  dkey_e = s P_e ([e chosen] dgate_e - sum_j P_j dgate_j)
//   sigmoid, renormalised:  w_j = s k_j / S, S = sum of the chosen keys
//                           dkey_j = (s / S) (dgate_j - sum_i (k_i / S) dgate_i)
//   sigmoid, raw:           dkey_j = s dgate_j
// and the logit gradient is dkey (softmax: the key is logit + bias) or dkey k (1 - k)
// (sigmoid: the key is sigma(logit)).
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace moe {
namespace {

constexpr int kWaves = 4;    // tokens per workgroup
constexpr int U = 4;         // 16-byte vectors per lane and row in one pass

// compact the token's local slots (slot order kept): rows, weights and slot indices into the
// wave's LDS lists; returns their number
__device__ __forceinline__ int compact_slots(const int32_t* slot_row, const float* topk_w, int64_t t, int k,
                                             int64_t cap, int lane, int* s_row, float* s_w, int* s_slot) {
  int r = -1;
  float wj = 0.f;
  if (lane < k) {
    r = slot_row[t * k + lane];
    if (r >= cap) r = -1;
    if (topk_w) wj = topk_w[t * k + lane];
  }
  const uint64_t act = __ballot(r >= 0);
  if (r >= 0) {
    const int pos = __popcll(act & ((1ull << lane) - 1ull));
    s_row[pos] = r;
    s_w[pos] = wj;
    s_slot[pos] = lane;
  }
  __builtin_amdgcn_wave_barrier();
  return __popcll(act);
}

__device__ __forceinline__ float bf_lo(uint32_t v) { return bf16_to_f32(v & 0xffffu); }
__device__ __forceinline__ float bf_hi(uint32_t v) { return bf16_to_f32(v >> 16); }

// dgate and dy_perm of one token per wave
__global__ __launch_bounds__(64 * kWaves) void k_combine_bwd(CombineBwdProblem p) {
  __shared__ int s_row[kWaves][16];
  __shared__ float s_w[kWaves][16];
  __shared__ int s_slot[kWaves][16];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t t = (int64_t)blockIdx.x * kWaves + wv;
  if (t >= p.T) return;                                   // wave-uniform
  const int k = p.top_k;
  const int nact = compact_slots(p.slot_row, p.topk_w, t, k, p.cap, lane, s_row[wv], s_w[wv], s_slot[wv]);
  // slots without a local row get a zero gate gradient
  if (lane < k) {
    const int r = p.slot_row[t * k + lane];
    if (r < 0 || r >= p.cap) p.dgate[t * k + lane] = 0.f;
  }
  if (nact == 0) return;
  int rows[16];
  float w[16];
#pragma unroll
  for (int a = 0; a < 16; ++a) {
    rows[a] = a < nact ? __builtin_amdgcn_readfirstlane(s_row[wv][a]) : 0;
    w[a] = a < nact ? __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(s_w[wv][a]))) : 0.f;
  }
  float part[16];
#pragma unroll
  for (int a = 0; a < 16; ++a) part[a] = 0.f;

  const int nvec = p.d / 8;
  const bf16_t* grow = p.dout + t * p.d;
  for (int v0 = 0; v0 < nvec; v0 += 64 * U) {
    u32x4 g[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = v0 + u * 64 + lane;
      g[u] = v < nvec ? ld16(grow + v * 8) : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int a = 0; a < 16; ++a) {
      if (a >= nact) continue;                            // wave-uniform
      const bf16_t* yrow = p.y_perm + (int64_t)rows[a] * p.d;
      bf16_t* drow = p.dy_perm + (int64_t)rows[a] * p.d;
      u32x4 y[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int v = v0 + u * 64 + lane;
        y[u] = v < nvec ? ld16(yrow + v * 8) : u32x4{0, 0, 0, 0};
      }
      float s = part[a];
#pragma unroll
      for (int u = 0; u < U; ++u) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          s += bf_lo(g[u][e]) * bf_lo(y[u][e]);
          s += bf_hi(g[u][e]) * bf_hi(y[u][e]);
        }
        const int v = v0 + u * 64 + lane;
        if (v < nvec) {
          u32x4 o;
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = pack_bf16x2(w[a] * bf_lo(g[u][e]), w[a] * bf_hi(g[u][e]));
          st16(drow + v * 8, o);
        }
      }
      part[a] = s;
    }
  }
#pragma unroll
  for (int a = 0; a < 16; ++a) {
    if (a < nact) {
      const float s = wave_sum(part[a]);
      if (lane == 0) p.dgate[t * k + s_slot[wv][a]] = s;
    }
  }
}

// dlogits [T, E] (bf16) of one token per wave; lane l owns experts [PL l, PL l + PL)
template <int PL>
__global__ __launch_bounds__(64 * kWaves) void k_gate_bwd(GateBwdProblem p) {
  __shared__ float s_key[kWaves][64 * PL];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t t = (int64_t)blockIdx.x * kWaves + w;
  if (blockIdx.x == 0) {
    if (threadIdx.x == 0 && p.seg) {
      p.seg[0] = 0;                                        // one row segment [0, T)
      p.seg[1] = (int32_t)p.T;
    }
    // token chunks of the router weight gradient's K split
    if (p.segk && (int)threadIdx.x <= p.nsegk)
      p.segk[threadIdx.x] = (int32_t)min((int64_t)threadIdx.x * p.segk_rows, p.T);
  }
  if (t >= p.T) return;                                   // wave-uniform
  const int E = p.E, k = p.top_k;
  const int e0 = lane * PL;
  const float s = p.routed_scale;

  // the forward's float32 keys: the K-chunk partials added in chunk order, then bias or sigmoid
  float key[PL];
#pragma unroll
  for (int j = 0; j < PL; ++j) key[j] = 0.f;
  const float* row0 = p.logits + t * E;
  for (int c = 0; c < p.nsplit; ++c) {
    const float* row = row0 + c * p.split_stride;
#pragma unroll
    for (int j = 0; j < PL; ++j) key[j] += (e0 + j < E) ? row[e0 + j] : 0.f;
  }
#pragma unroll
  for (int j = 0; j < PL; ++j) {
    const int e = e0 + j;
    if (e < E) {
      const float L = key[j];
      key[j] = (p.gate == 0) ? (p.bias ? L + p.bias[e] : L) : 1.0f / (1.0f + expf(-L));
    }
    s_key[w][e] = key[j];
  }
  __builtin_amdgcn_wave_barrier();

  // lane j < k: slot j's expert, its key and its gate gradient
  int idx = 0;
  float kc = 0.f, dg = 0.f;
  if (lane < k) {
    idx = min(max(p.topk_idx[t * k + lane], 0), E - 1);
    kc = s_key[w][idx];
    dg = p.dgate[t * k + lane];
  }
  const bool chosen = lane < k;
  float dl = 0.f;                                         // logit gradient of slot `lane`
  float m = 0.f, den = 1.f, inner = 0.f;                  // softmax over all E: shift, normaliser, inner
  const bool full_softmax = p.gate == 0 && !p.renormalize;
  if (full_softmax) {
    float mm = -INFINITY;
#pragma unroll
    for (int j = 0; j < PL; ++j)
      if (e0 + j < E) mm = fmaxf(mm, key[j]);
    m = wave_max(mm);
    float part = 0.f;
#pragma unroll
    for (int j = 0; j < PL; ++j)
      if (e0 + j < E) part += expf(key[j] - m);
    den = wave_sum(part);
    inner = wave_sum(chosen ? expf(kc - m) / den * dg : 0.f);
  } else if (p.gate == 0) {
    // renormalised softmax over the chosen keys
    const float mc = wave_max(chosen ? kc : -INFINITY);
    const float ev = chosen ? expf(kc - mc) : 0.f;
    const float dsum = wave_sum(ev);
    const float pj = ev / dsum;
    const float in = wave_sum(chosen ? pj * dg : 0.f);
    dl = chosen ? s * pj * (dg - in) : 0.f;
  } else if (p.renormalize) {
    const float S = wave_sum(chosen ? kc : 0.f);
    const float in = wave_sum(chosen ? (kc / S) * dg : 0.f);
    dl = chosen ? (s / S) * (dg - in) * kc * (1.0f - kc) : 0.f;
  } else {
    dl = chosen ? s * dg * kc * (1.0f - kc) : 0.f;
  }

  // each lane assembles its PL entries of the row
  float out[PL];
#pragma unroll
  for (int j = 0; j < PL; ++j) {
    out[j] = 0.f;
    if (full_softmax && e0 + j < E) out[j] = -s * (expf(key[j] - m) / den) * inner;
  }
  for (int r = 0; r < k; ++r) {
    const int er = __builtin_amdgcn_readlane(idx, r);
    const unsigned off = (unsigned)(er - e0);
    if (off < (unsigned)PL) {
      float add;
      if (full_softmax) {
        const float dgr = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(dg), r));
        add = s * (expf(s_key[w][er] - m) / den) * dgr;
      } else {
        add = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(dl), r));
      }
#pragma unroll
      for (int j = 0; j < PL; ++j)
        if ((unsigned)j == off) out[j] += add;
    }
  }
  bf16_t* orow = p.dlogits + t * E;
#pragma unroll
  for (int j = 0; j < PL; ++j)
    if (e0 + j < E) orow[e0 + j] = (bf16_t)f32_to_bf16(out[j]);
}

// dx[t] = bf16( sum over local slots (slot order) of dx_perm[row] + extra0[t] + extra1[t] )
__global__ __launch_bounds__(64 * kWaves) void k_unpermute_sum(UnpermuteSumProblem p) {
  __shared__ int s_row[kWaves][16];
  __shared__ float s_w[kWaves][16];
  __shared__ int s_slot[kWaves][16];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t t = (int64_t)blockIdx.x * kWaves + wv;
  if (t >= p.T) return;                                   // wave-uniform
  const int nact = compact_slots(p.slot_row, nullptr, t, p.top_k, p.cap, lane, s_row[wv], s_w[wv], s_slot[wv]);
  int rows[16];
#pragma unroll
  for (int a = 0; a < 16; ++a) rows[a] = a < nact ? __builtin_amdgcn_readfirstlane(s_row[wv][a]) : 0;
  const int nvec = p.d / 8;
  for (int v0 = 0; v0 < nvec; v0 += 64 * U) {
    float acc[U][8];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[u][e] = 0.f;
    auto add_row = [&](const bf16_t* row) {
      u32x4 y[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int v = v0 + u * 64 + lane;
        y[u] = v < nvec ? ld16(row + v * 8) : u32x4{0, 0, 0, 0};
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[u][2 * e] += bf_lo(y[u][e]);
          acc[u][2 * e + 1] += bf_hi(y[u][e]);
        }
    };
    // two rows' loads in flight at a time; the additions keep the slot order (then extra0, extra1)
    auto add_two = [&](const bf16_t* r0, const bf16_t* r1) {
      u32x4 y0[U], y1[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int v = v0 + u * 64 + lane;
        y0[u] = v < nvec ? ld16(r0 + v * 8) : u32x4{0, 0, 0, 0};
        y1[u] = v < nvec ? ld16(r1 + v * 8) : u32x4{0, 0, 0, 0};
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[u][2 * e] += bf_lo(y0[u][e]);
          acc[u][2 * e + 1] += bf_hi(y0[u][e]);
        }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[u][2 * e] += bf_lo(y1[u][e]);
          acc[u][2 * e + 1] += bf_hi(y1[u][e]);
        }
    };
    int a = 0;
#pragma unroll
    for (int pr = 0; pr < 8; ++pr) {
      if (a + 1 >= nact) break;
      add_two(p.rows + (int64_t)rows[a] * p.d, p.rows + (int64_t)rows[a + 1] * p.d);
      a += 2;
    }
    if (a < nact) {
      // an odd last row pairs with the first extra row when there is one
      if (p.extra0) {
        add_two(p.rows + (int64_t)rows[a] * p.d, p.extra0 + t * p.d);
        if (p.extra1) add_row(p.extra1 + t * p.d);
      } else {
        add_row(p.rows + (int64_t)rows[a] * p.d);
        if (p.extra1) add_row(p.extra1 + t * p.d);
      }
    } else if (p.extra0 && p.extra1) {
      add_two(p.extra0 + t * p.d, p.extra1 + t * p.d);
    } else {
      if (p.extra0) add_row(p.extra0 + t * p.d);
      if (p.extra1) add_row(p.extra1 + t * p.d);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = v0 + u * 64 + lane;
      if (v >= nvec) continue;
      u32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = pack_bf16x2(acc[u][2 * e], acc[u][2 * e + 1]);
      st16(p.out + t * p.d + v * 8, o);
    }
  }
}

// out = bf16 of the float32 partials summed in order, four values per thread
__global__ __launch_bounds__(256) void k_sum_partials(const float* parts, int nparts, int64_t n4, bf16_t* out) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256) {
    f32x4 acc = reinterpret_cast<const f32x4*>(parts)[i];
    for (int s = 1; s < nparts; ++s) {
      const f32x4 v = reinterpret_cast<const f32x4*>(parts + (int64_t)s * n4 * 4)[i];
      acc[0] += v[0];
      acc[1] += v[1];
      acc[2] += v[2];
      acc[3] += v[3];
    }
    uint2 o;
    o.x = pack_bf16x2(acc[0], acc[1]);
    o.y = pack_bf16x2(acc[2], acc[3]);
    *reinterpret_cast<uint2*>(out + 4 * i) = o;
  }
}

template <int PL>
hipError_t launch_gate_bwd_pl(const GateBwdProblem& p, hipStream_t stream) {
  const unsigned blocks = (unsigned)((p.T + kWaves - 1) / kWaves);
  hipLaunchKernelGGL(k_gate_bwd<PL>, dim3(blocks > 0 ? blocks : 1), dim3(64 * kWaves), 0, stream, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_combine_bwd(const CombineBwdProblem& p, hipStream_t stream) {
  if (p.top_k < 1 || p.top_k > 16 || p.d % 8) return hipErrorInvalidValue;
  const unsigned blocks = (unsigned)((p.T + kWaves - 1) / kWaves);
  hipLaunchKernelGGL(k_combine_bwd, dim3(blocks), dim3(64 * kWaves), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_sum_partials(const float* parts, int nparts, int64_t n, bf16_t* out, hipStream_t stream) {
  if (nparts < 1 || n % 4) return hipErrorInvalidValue;
  const int64_t n4 = n / 4;
  const int64_t b = (n4 + 255) / 256;
  hipLaunchKernelGGL(k_sum_partials, dim3((unsigned)(b < 4096 ? (b > 0 ? b : 1) : 4096)), dim3(256), 0, stream, parts,
                     nparts, n4, out);
  return hipGetLastError();
}

hipError_t launch_gate_bwd(const GateBwdProblem& p, hipStream_t stream) {
  if (p.nsplit < 1 || p.top_k < 1 || p.top_k > 16 || p.E < 1) return hipErrorInvalidValue;
  if (p.segk && (p.nsegk < 1 || p.nsegk >= 64 * kWaves || p.segk_rows < 1)) return hipErrorInvalidValue;
  const int pl = (p.E + 63) / 64;
  if (pl <= 1) return launch_gate_bwd_pl<1>(p, stream);
  if (pl <= 2) return launch_gate_bwd_pl<2>(p, stream);
  if (pl <= 4) return launch_gate_bwd_pl<4>(p, stream);
  if (pl <= 8) return launch_gate_bwd_pl<8>(p, stream);
  if (pl <= 16) return launch_gate_bwd_pl<16>(p, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_unpermute_sum(const UnpermuteSumProblem& p, hipStream_t stream) {
  if (p.top_k < 1 || p.top_k > 16 || p.d % 8) return hipErrorInvalidValue;
  const unsigned blocks = (unsigned)((p.T + kWaves - 1) / kWaves);
  hipLaunchKernelGGL(k_unpermute_sum, dim3(blocks), dim3(64 * kWaves), 0, stream, p);
  return hipGetLastError();
}

}  // namespace moe
