// Gate-weighted combine: one wavefront per token, owner computes (no atomics); and the
// clear / rounding passes of the combine folded into the down-projection.
//
//   out[t] = bf16( sum_j topk_w[t,j] * y_perm[slot_row[t,j]]  (+ shared_y[t]) )
//
// float32 accumulation in slot order, the shared row last, one round-to-nearest-even.
// The token's local slots are compacted first (lane j holds slot j; a ballot gives each
// local slot its position), so the row loop runs over local rows only, with no branch per
// slot.  Each lane streams 16-byte vectors; per pass the shared row's loads are issued first
// and the expert rows' loads two rows at a time, so several rows are in flight per wave.
#include "common.hpp"
#include "kernels.hpp"

namespace moe {
namespace {

constexpr int kWaves = 4;    // tokens per workgroup
constexpr int U = 4;         // 16-byte vectors per lane and row in one pass

__device__ __forceinline__ void fma_row(float (&acc)[U][8], const u32x4 (&y)[U], float w) {
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[u][2 * e] += w * bf16_to_f32(y[u][e] & 0xffffu);
      acc[u][2 * e + 1] += w * bf16_to_f32(y[u][e] >> 16);
    }
}

__global__ __launch_bounds__(64 * kWaves) void k_combine(CombineProblem p) {
  __shared__ int s_row[kWaves][16];
  __shared__ float s_w[kWaves][16];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t t = (int64_t)blockIdx.x * kWaves + wv;
  if (t >= p.T) return;                                   // wave-uniform
  const int k = p.top_k;

  // compact the local slots, keeping slot order
  int r = -1;
  float wj = 0.f;
  if (lane < k) {
    r = p.slot_row[t * k + lane];
    if (r >= p.cap) r = -1;
    wj = p.topk_w[t * k + lane];
  }
  const uint64_t act = __ballot(r >= 0);
  const int nact = __popcll(act);
  if (r >= 0) {
    const int pos = __popcll(act & ((1ull << lane) - 1ull));
    s_row[wv][pos] = r;
    s_w[wv][pos] = wj;
  }
  __builtin_amdgcn_wave_barrier();
  int rows[16];
  float w[16];
#pragma unroll
  for (int a = 0; a < 16; ++a) {
    rows[a] = a < nact ? __builtin_amdgcn_readfirstlane(s_row[wv][a]) : 0;
    w[a] = a < nact ? __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(s_w[wv][a]))) : 0.f;
  }

  const int nvec = p.d / 8;
  const bf16_t* srow = p.shared_y ? p.shared_y + t * p.d : nullptr;
  for (int v0 = 0; v0 < nvec; v0 += 64 * U) {
    u32x4 sy[U];
    if (srow) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int v = v0 + u * 64 + lane;
        sy[u] = v < nvec ? ld16(srow + v * 8) : u32x4{0, 0, 0, 0};
      }
    }
    float acc[U][8];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[u][e] = 0.f;
#pragma unroll
    for (int a = 0; a < 16; a += 2) {
      if (a >= nact) break;
      const bool two = a + 1 < nact;
      const bf16_t* y0 = p.y_perm + (int64_t)rows[a] * p.d;
      const bf16_t* y1 = p.y_perm + (int64_t)rows[two ? a + 1 : a] * p.d;
      u32x4 ya[U], yb[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int v = v0 + u * 64 + lane;
        ya[u] = v < nvec ? ld16(y0 + v * 8) : u32x4{0, 0, 0, 0};
      }
      if (two) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int v = v0 + u * 64 + lane;
          yb[u] = v < nvec ? ld16(y1 + v * 8) : u32x4{0, 0, 0, 0};
        }
      }
      fma_row(acc, ya, w[a]);
      if (two) fma_row(acc, yb, w[a + 1]);
    }
    if (srow) {
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[u][2 * e] += bf16_to_f32(sy[u][e] & 0xffffu);
          acc[u][2 * e + 1] += bf16_to_f32(sy[u][e] >> 16);
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

// The float32 accumulator of the combine folded into the down-projection: cleared before
// the GEMM, rounded to bf16 after it (16-byte loads and stores, grid-stride).
__global__ __launch_bounds__(256) void k_zero_f32(float* acc, int64_t n4) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256)
    reinterpret_cast<f32x4*>(acc)[i] = f32x4{0.f, 0.f, 0.f, 0.f};
}

__global__ __launch_bounds__(256) void k_round_bf16(const float* acc, bf16_t* out, int64_t n8) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n8; i += (int64_t)gridDim.x * 256) {
    const f32x4 a = reinterpret_cast<const f32x4*>(acc)[2 * i];
    const f32x4 b = reinterpret_cast<const f32x4*>(acc)[2 * i + 1];
    u32x4 o;
    o[0] = pack_bf16x2(a[0], a[1]);
    o[1] = pack_bf16x2(a[2], a[3]);
    o[2] = pack_bf16x2(b[0], b[1]);
    o[3] = pack_bf16x2(b[2], b[3]);
    st16(out + 8 * i, o);
  }
}

unsigned stream_blocks(int64_t items) {
  const int64_t b = (items + 255) / 256;
  return (unsigned)(b < 8192 ? (b > 0 ? b : 1) : 8192);   // 32 workgroups per CU at most
}

}  // namespace

hipError_t launch_zero_f32(float* acc, int64_t n, hipStream_t stream) {
  if (n % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_zero_f32, dim3(stream_blocks(n / 4)), dim3(256), 0, stream, acc, n / 4);
  return hipGetLastError();
}

hipError_t launch_round_bf16(const float* acc, bf16_t* out, int64_t n, hipStream_t stream) {
  if (n % 8) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_round_bf16, dim3(stream_blocks(n / 8)), dim3(256), 0, stream, acc, out, n / 8);
  return hipGetLastError();
}

hipError_t launch_combine(const CombineProblem& p, hipStream_t stream) {
  const unsigned blocks = (unsigned)((p.T + kWaves - 1) / kWaves);
  hipLaunchKernelGGL(k_combine, dim3(blocks), dim3(64 * kWaves), 0, stream, p);
  return hipGetLastError();
}

}  // namespace moe
