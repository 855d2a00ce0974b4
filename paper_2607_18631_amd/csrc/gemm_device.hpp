// Device helpers shared by the grouped GEMMs (forward and backward): slice copies straight
// into LDS, wait / barrier primitives, the K-major LDS swizzle, a block-wide scan and the
// XCD-aware first tile of a persistent workgroup.
#pragma once
#include <type_traits>

#include "common.hpp"

namespace moe {

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"I"(N) : "memory");
}
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
__device__ __forceinline__ void raw_barrier() { asm volatile("s_barrier" ::: "memory"); }

// 16-byte direct-to-LDS copy of one wave instruction: lane i fetches `src` (its own
// address) into bytes [16 i, 16 i + 16) after the wave-uniform LDS address `dst`.
__device__ __forceinline__ void dma16(const bf16_t* src, bf16_t* dst) {
  __builtin_amdgcn_global_load_lds(src, dst, 16, 0, 0);
}

// The same copy written as inline assembly, from a wave-uniform base `sbase` plus the lane's
// 32-bit byte offset `voff`: no 64-bit per-lane address arithmetic per copy, and only the
// 32-bit offsets stay live across a K loop.  Also for kernels that read LDS with
// ds_read_b64_tr_b16: the compiler makes every such read wait for all direct-to-LDS copies it
// knows of (vmcnt(0)), which would serialise each slice's copies with the next slice's MFMAs.
// Copies issued this way are invisible to it; the kernel orders them itself (explicit vmcnt
// counts and barriers).  M0 carries the LDS address; the asm declares M0 clobbered, so the
// compiler keeps nothing of its own there across it.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16_sv(const char* sbase, uint32_t voff, bf16_t* dst) {
  const uint32_t lds = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) bf16_t*)(dst);
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "s"(lds)
               : "memory", "m0");
}
#pragma clang diagnostic pop

template <int BK>
struct Swz {
  static constexpr int CPR = BK / 8;            // 16-byte chunks per row
  static constexpr int RPG = 16 / CPR;          // rows per 256-byte bank cycle
  __device__ static __forceinline__ int f(int row) { return (row / RPG) % CPR; }
  __device__ static __forceinline__ int off(int row, int chunk) { return row * BK + ((chunk ^ f(row)) << 3); }
};

// Block-wide exclusive scan of one int per thread (NTH threads); returns the block total.
template <int NTH>
__device__ int block_exclusive_scan(int v, int* s_tmp, int& excl) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int n = __shfl_up(inc, o, 64);
    if (lane >= o) inc += n;
  }
  if (lane == 63) s_tmp[wave] = inc;
  __syncthreads();
  int wbase = 0, total = 0;
#pragma unroll
  for (int w = 0; w < NTH / 64; ++w) {
    int t = s_tmp[w];
    if (w < wave) wbase += t;
    total += t;
  }
  excl = wbase + inc - v;
  __syncthreads();
  return total;
}

// Workgroup b's first tile: adjacent tiles go to workgroups of one XCD (b runs on XCD b % 8).
__device__ __forceinline__ int first_tile_slot() {
  const int G = gridDim.x;
  return (G % 8 == 0) ? (int)(blockIdx.x % 8) * (G / 8) + (int)(blockIdx.x / 8) : (int)blockIdx.x;
}

// Instruction-scheduler directives for one MFMA K-step: an MFMA first, then the next
// step's LDS reads two at a time between MFMAs, then the remaining MFMAs.
template <int REM>
__device__ __forceinline__ void sched_read_pairs() {
  if constexpr (REM > 0) {
    __builtin_amdgcn_sched_group_barrier(0x100, REM >= 2 ? 2 : 1, 0);   // DS read(s)
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                  // one MFMA
    sched_read_pairs<REM - 2>();
  }
}
template <int NR, int NMF>
__device__ __forceinline__ void sched_step() {
  if constexpr (NMF >= (NR + 1) / 2 + 1) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    sched_read_pairs<NR>();
    if constexpr (NMF - (NR + 1) / 2 - 1 > 0)
      __builtin_amdgcn_sched_group_barrier(0x008, NMF - (NR + 1) / 2 - 1, 0);
  }
  __builtin_amdgcn_sched_barrier(0);
}

// f(std::integral_constant<int, k>) with k = min(n, N) (n >= 0)
template <int N, class F>
__device__ __forceinline__ void with_count(int n, F&& f) {
  if constexpr (N == 0) {
    f(std::integral_constant<int, 0>{});
  } else {
    if (n >= N) f(std::integral_constant<int, N>{});
    else with_count<N - 1>(n, f);
  }
}

}  // namespace moe
