// Bandwidth probes of the benchmark (libmoe_probe.so, not part of the MoE library): a read-only
// stream, the practical HBM read ceiling the layer's HBM-bound kernels are compared with.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

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
