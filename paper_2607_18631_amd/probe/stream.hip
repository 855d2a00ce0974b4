// Probes of the benchmark (libmoe_probe.so, not part of the MoE library): a read-only stream, the
// practical HBM read ceiling the layer's HBM-bound kernels are compared with, and a loop of
// independent bf16 MFMAs on register operands, the practical MFMA ceiling under full load (the
// clock the part sustains with every matrix pipe busy, below the nominal 2.4 GHz).
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Every lane reads 16-byte vectors at a grid stride, U in flight, and folds them with XOR; one
// 4-byte store per wave keeps the loads alive.
__global__ __launch_bounds__(256) void k_read_stream(const u32x4* src, int64_t n, uint32_t* sink) {
  constexpr int U = 8;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  uint32_t acc = 0;
  for (int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i0 < n; i0 += U * stride) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = i0 + u * stride;
      v[u] = i < n ? __builtin_nontemporal_load(src + i) : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (int o = 32; o >= 1; o >>= 1) acc ^= __shfl_xor(acc, o, 64);
  if ((threadIdx.x & 63) == 0) sink[(blockIdx.x * blockDim.x + threadIdx.x) >> 6] = acc;
}

constexpr int kMfmaChains = 4;         // independent accumulators per wave
constexpr int kMfmaBlocks = 256 * 2;   // two workgroups of 4 waves per compute unit (2 waves per SIMD)

// Each wave issues iters x kMfmaChains v_mfma_f32_32x32x16_bf16 on fixed register operands (bf16
// values from a hash of the lane, so the multipliers see varied data), then stores one float per
// lane so that the loop is kept.
__global__ __launch_bounds__(256) void k_mfma_loop(int iters, float* sink) {
  const uint32_t lane = threadIdx.x;
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t h = (lane * 2654435761u) ^ (uint32_t)(i * 40503u);
    a[i] = (__bf16)((float)((h >> 8) & 0xff) * (1.0f / 256.0f) - 0.5f);
    b[i] = (__bf16)((float)((h >> 16) & 0xff) * (1.0f / 256.0f) - 0.5f);
  }
  f32x16 acc[kMfmaChains];
#pragma unroll
  for (int c = 0; c < kMfmaChains; ++c)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[c][i] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kMfmaChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  float r = 0.f;
#pragma unroll
  for (int c = 0; c < kMfmaChains; ++c)
#pragma unroll
    for (int i = 0; i < 16; ++i) r += acc[c][i];
  sink[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = r;
}

}  // namespace

// Reads `bytes` (a multiple of 16) from the device buffer `src`; `sink` holds at least
// probe_read_sink_words() 32-bit words.  Returns a hipError_t.
extern "C" int probe_read_stream(const void* src, int64_t bytes, void* sink, void* stream) {
  if (!src || !sink || bytes <= 0 || bytes % 16) return (int)hipErrorInvalidValue;
  const int blocks = 256 * 8;   // 8 workgroups of 4 waves per compute unit
  hipLaunchKernelGGL(k_read_stream, dim3(blocks), dim3(256), 0, reinterpret_cast<hipStream_t>(stream),
                     static_cast<const u32x4*>(src), bytes / 16, static_cast<uint32_t*>(sink));
  return (int)hipGetLastError();
}

extern "C" int64_t probe_read_sink_words(void) { return 256 * 8 * 4; }

// Runs the MFMA loop: probe_mfma_blocks() workgroups of 256 threads, each wave issuing iters x 4
// MFMAs of 32 x 32 x 16 (32,768 flop each); `sink` holds probe_mfma_blocks() * 256 floats.
// Returns a hipError_t.
extern "C" int probe_mfma_loop(int iters, void* sink, void* stream) {
  if (!sink || iters < 1) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(k_mfma_loop, dim3(kMfmaBlocks), dim3(256), 0, reinterpret_cast<hipStream_t>(stream), iters,
                     static_cast<float*>(sink));
  return (int)hipGetLastError();
}

extern "C" int64_t probe_mfma_blocks(void) { return kMfmaBlocks; }

// Flops of one probe_mfma_loop call.
extern "C" double probe_mfma_flops(int iters) { return (double)kMfmaBlocks * 4 * iters * kMfmaChains * 32768.0; }
