// Gate-weighted combine: one wavefront per token, owner computes (no atomics).
//
//   out[t] = bf16( sum_j topk_w[t,j] * y_perm[slot_row[t,j]]  (+ shared_y[t]) )
//
// float32 accumulation in slot order, the shared row last, one round-to-nearest-even.
// The slot rows and gates are wave-uniform; each lane streams 16-byte vectors of the
// k_local expert rows, so every row read is a fully coalesced 128-byte-per-8-lanes burst.
#include "common.hpp"
#include "kernels.hpp"

namespace moe {
namespace {

__global__ __launch_bounds__(256) void k_combine(CombineProblem p) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= p.T) return;
  const int k = p.top_k;
  int rows[16];
  float w[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    rows[j] = -1;
    w[j] = 0.f;
    if (j < k) {
      rows[j] = p.slot_row[t * k + j];
      if (rows[j] >= p.cap) rows[j] = -1;
      w[j] = p.topk_w[t * k + j];
    }
  }
  constexpr int U = 4;                       // 16-byte vectors per lane in flight per row
  const int nvec = p.d / 8;
  for (int v0 = 0; v0 < nvec; v0 += 64 * U) {
    float acc[U][8];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[u][e] = 0.f;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if (rows[j] < 0) continue;
      const bf16_t* yrow = p.y_perm + (int64_t)rows[j] * p.d;
      u32x4 y[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int v = v0 + u * 64 + lane;
        y[u] = v < nvec ? ld16(yrow + v * 8) : u32x4{0, 0, 0, 0};
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[u][2 * e] += w[j] * bf16_to_f32(y[u][e] & 0xffffu);
          acc[u][2 * e + 1] += w[j] * bf16_to_f32(y[u][e] >> 16);
        }
    }
    if (p.shared_y) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int v = v0 + u * 64 + lane;
        if (v >= nvec) continue;
        const u32x4 sy = ld16(p.shared_y + t * p.d + v * 8);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[u][2 * e] += bf16_to_f32(sy[e] & 0xffffu);
          acc[u][2 * e + 1] += bf16_to_f32(sy[e] >> 16);
        }
      }
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

}  // namespace

hipError_t launch_combine(const CombineProblem& p, hipStream_t stream) {
  const unsigned blocks = (unsigned)((p.T + 3) / 4);
  hipLaunchKernelGGL(k_combine, dim3(blocks), dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace moe
