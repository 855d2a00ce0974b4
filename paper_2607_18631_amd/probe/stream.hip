// Probes of the benchmark (libmoe_probe.so, not part of the MoE library): a read-only stream, the
// practical HBM read ceiling the layer's HBM-bound kernels are compared with; a loop of
// independent bf16 MFMAs on register operands, the practical MFMA ceiling under full load (the
// clock the part sustains with every matrix pipe busy, below the nominal 2.4 GHz); and an LDS read
// stream, the LDS bandwidth the GEMM's fragment reads and slice copies share.
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

constexpr int kLdsBlocks = 256 * 2;    // two workgroups of 4 waves (64 KB of LDS each) per compute unit
constexpr int kLdsBatch = 8;           // ds_read_b128 per batch; at most 15 in flight (lgkmcnt)

// Each wave reads iters x kLdsBatch 1 KB rows of its workgroup's 64 KB LDS array with ds_read_b128
// (64 lanes x 16 consecutive bytes: no bank conflicts), at most 15 reads in flight.  The reads
// are inline asm so the compiler keeps every one; the last batch is folded into `sink`.  Wave 0
// of each workgroup stores the shader-clock cycles (s_memtime) and the fixed 100 MHz ticks
// (s_memrealtime) its loop took, so the host gets bytes per clock and the clock itself.
__global__ __launch_bounds__(256) void k_lds_read(int iters, uint32_t* sink, uint64_t* cycles) {
  __shared__ u32x4 buf[4096];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = tid; i < 4096; i += 256) buf[i] = u32x4{(uint32_t)i, (uint32_t)i * 3u, (uint32_t)i * 5u, (uint32_t)i * 7u};
  __syncthreads();
  const uint32_t addr = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) u32x4*)(buf + wave * 64 + lane);
  const uint64_t c0 = __builtin_amdgcn_s_memtime(), r0 = __builtin_amdgcn_s_memrealtime();
  u32x4 v0, v1, v2, v3, v4, v5, v6, v7;
  for (int it = 0; it < iters; ++it) {
    asm volatile(
        "ds_read_b128 %0, %8\n\t"
        "ds_read_b128 %1, %8 offset:4096\n\t"
        "ds_read_b128 %2, %8 offset:8192\n\t"
        "ds_read_b128 %3, %8 offset:12288\n\t"
        "ds_read_b128 %4, %8 offset:16384\n\t"
        "ds_read_b128 %5, %8 offset:20480\n\t"
        "ds_read_b128 %6, %8 offset:24576\n\t"
        "ds_read_b128 %7, %8 offset:28672\n\t"
        "s_waitcnt lgkmcnt(7)"
        : "=&v"(v0), "=&v"(v1), "=&v"(v2), "=&v"(v3), "=&v"(v4), "=&v"(v5), "=&v"(v6), "=&v"(v7)
        : "v"(addr)
        : "memory");
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  const uint64_t c1 = __builtin_amdgcn_s_memtime(), r1 = __builtin_amdgcn_s_memrealtime();
  const u32x4 x = v0 ^ v1 ^ v2 ^ v3 ^ v4 ^ v5 ^ v6 ^ v7;
  sink[(int64_t)blockIdx.x * 256 + tid] = x.x ^ x.y ^ x.z ^ x.w;
  if (tid == 0) {
    cycles[2 * blockIdx.x] = c1 - c0;
    cycles[2 * blockIdx.x + 1] = r1 - r0;
  }
}

}  // namespace

// Runs the LDS read loop: probe_lds_blocks() workgroups of 256 threads, each wave reading
// iters x 8 KB of LDS.  `sink` holds probe_lds_blocks() * 256 words, `cycles` 2 * probe_lds_blocks()
// 64-bit words (per workgroup: shader-clock cycles, then 100 MHz ticks, of wave 0's loop).
// Returns a hipError_t.
extern "C" int probe_lds_read(int iters, void* sink, void* cycles, void* stream) {
  if (!sink || !cycles || iters < 1) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(k_lds_read, dim3(kLdsBlocks), dim3(256), 0, reinterpret_cast<hipStream_t>(stream), iters,
                     static_cast<uint32_t*>(sink), static_cast<uint64_t*>(cycles));
  return (int)hipGetLastError();
}

extern "C" int64_t probe_lds_blocks(void) { return kLdsBlocks; }

// LDS bytes one probe_lds_read call reads.
extern "C" double probe_lds_bytes(int iters) { return (double)kLdsBlocks * 4 * iters * kLdsBatch * 1024.0; }

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
