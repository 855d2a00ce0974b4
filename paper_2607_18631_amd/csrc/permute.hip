// Histogram, prefix scan and stable permutation of the local (token, expert) slots.
//
// Tokens are cut into chunks of 64 (one wavefront).  Four launches:
//   k_chunk_count  per chunk, how many of its slots go to each local expert
//   k_chunk_scan   per expert, exclusive scan of the chunk counts over chunks, and
//                  the expert total (counts[e])
//   k_rank         per chunk: the offsets (exclusive scan of counts, the monotone
//                  [E_local+1] array), each slot's rank among the chunk's earlier slots
//                  of the same expert (slot columns spread over the waves), hence its row
//                      row = offsets[e] + chunk_base[c][e] + rank,
//                  then row_token / slot_row (and the gate of each row when asked)
//   k_gather       per token: the bit-exact copy of the token row to each of its local
//                  rows (read once, written k_local times, 16-byte vectors); skipped when
//                  the caller's GEMM reads the token rows through row_token itself
//
// Masked-decode layout (expert capacity C > 0): expert e's rows are e * C + rank for the
// ranks below C; later slots are dropped (slot_row = -1) and offsets[e] = e * C.
//
// The in-chunk rank uses wavefront ballots instead of atomics, so the order inside an
// expert is ascending token (a stable counting sort) and run-to-run identical: for every
// slot column j' and every bit b of the local expert id, one ballot gives the lanes whose
// slot j' has bit b set; AND-ing the matching ballots (or their complements) yields the
// lanes whose slot j' holds exactly my expert, and the popcount below my lane is the rank.
#include <mutex>

#include "common.hpp"
#include "kernels.hpp"

namespace moe {
namespace {

constexpr int CH = 64;          // tokens per chunk = lanes of one wave

__global__ __launch_bounds__(64) void k_chunk_count(PermuteProblem p) {
  extern __shared__ int s_cnt[];   // [E_local]
  const int lane = threadIdx.x;
  for (int e = lane; e < p.E_local; e += 64) s_cnt[e] = 0;
  __syncthreads();
  const int64_t t = (int64_t)blockIdx.x * CH + lane;
  if (t < p.T) {
    for (int j = 0; j < p.top_k; ++j) {
      const int le = p.topk_idx[t * p.top_k + j] - p.e_begin;
      if (le >= 0 && le < p.E_local) atomicAdd(&s_cnt[le], 1);
    }
  }
  __syncthreads();
  int32_t* dst = p.blk_count + (int64_t)blockIdx.x * p.E_local;
  for (int e = lane; e < p.E_local; e += 64) dst[e] = s_cnt[e];
}

// one workgroup per local expert: exclusive scan of blk_count[:, e] over chunks
__global__ __launch_bounds__(256) void k_chunk_scan(PermuteProblem p, int nblk) {
  __shared__ int s_w[4];
  const int e = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int carry = 0;
  for (int b0 = 0; b0 < nblk; b0 += 256) {
    const int b = b0 + tid;
    const int v = b < nblk ? p.blk_count[(int64_t)b * p.E_local + e] : 0;
    int inc = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      int n = __shfl_up(inc, o, 64);
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
    if (b < nblk) p.blk_base[(int64_t)b * p.E_local + e] = carry + wbase + inc - v;
    carry += tot;
    __syncthreads();
  }
  if (tid == 0) p.counts[e] = carry;
}

// one workgroup per chunk: offsets (every workgroup; workgroup 0 publishes them), then the
// chunk's slots are ranked, wave w taking slot columns w, w + RW, ... (every wave forms the
// ballots of all columns, which are cheap; the per-slot rank work is split)
constexpr int RW = 8;                          // waves of the rank kernel
__global__ __launch_bounds__(64 * RW) void k_rank(PermuteProblem p) {
  extern __shared__ int s_off[];               // [E_local + 1]
  __shared__ int s_w[RW];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = blockIdx.x;
  const int E_local = p.E_local, k = p.top_k;

  // offsets = exclusive scan of counts
  {
    constexpr int PER = (1024 + 64 * RW - 1) / (64 * RW);   // threads x PER >= 1024 experts
    int v[PER], lsum = 0;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = tid * PER + i;
      v[i] = e < E_local ? p.counts[e] : 0;
      lsum += v[i];
    }
    int inc = lsum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      int n = __shfl_up(inc, o, 64);
      if (lane >= o) inc += n;
    }
    if (lane == 63) s_w[wave] = inc;
    __syncthreads();
    int run = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < RW; ++w) {
      if (w < wave) run += s_w[w];
      tot += s_w[w];
    }
    run += inc - lsum;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = tid * PER + i;
      if (e < E_local) s_off[e] = run;
      run += v[i];
    }
    if (tid == 0) s_off[E_local] = tot;
    __syncthreads();
    if (c == 0)
      for (int e = tid; e <= E_local; e += 64 * RW)
        p.offsets[e] = p.expert_capacity > 0 ? e * p.expert_capacity : s_off[e];
  }
  if (wave >= k) return;                       // wave-uniform

  // rank of each of my slots among the chunk's earlier slots of the same expert
  const int64_t t = (int64_t)c * CH + lane;
  const bool valid_t = t < p.T;
  int nbits = 0;
  while ((1 << nbits) < E_local) ++nbits;
  const int32_t* base = p.blk_base + (int64_t)c * E_local;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  constexpr int MINE = (16 + RW - 1) / RW;     // slot columns per wave (top_k <= 16)
  int myle[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    myle[j] = -1;
    if (j < k && valid_t) {
      const int le = p.topk_idx[t * k + j] - p.e_begin;
      myle[j] = (le >= 0 && le < E_local) ? le : -1;
    }
  }
  int rank[MINE];
#pragma unroll
  for (int m = 0; m < MINE; ++m) rank[m] = 0;
#pragma unroll
  for (int jp = 0; jp < 16; ++jp) {
    if (jp >= k) break;
    // lanes whose slot jp is local, and per bit the lanes whose slot jp has that bit set
    const int lej = myle[jp];
    const uint64_t vmask = __ballot(lej >= 0);
    uint64_t bal[10];
#pragma unroll
    for (int b = 0; b < 10; ++b) bal[b] = (b < nbits) ? __ballot(lej >= 0 && ((lej >> b) & 1)) : 0ull;
#pragma unroll
    for (int m = 0; m < MINE; ++m) {
      const int j = wave + m * RW;
      if (j >= k) break;
      const int le = myle[j];
      uint64_t msk = vmask;
#pragma unroll
      for (int b = 0; b < 10; ++b)
        if (b < nbits) msk &= ((le >> b) & 1) ? bal[b] : ~bal[b];
      rank[m] += __popcll(msk & below);
    }
  }
  if (!valid_t) return;
#pragma unroll
  for (int m = 0; m < MINE; ++m) {
    const int j = wave + m * RW;
    if (j >= k) break;
    int row = -1;
    if (myle[j] >= 0) {
      const int grank = base[myle[j]] + rank[m];             // rank inside the expert
      if (p.expert_capacity > 0)                             // masked-decode layout: drop past C
        row = grank < p.expert_capacity ? myle[j] * p.expert_capacity + grank : -1;
      else
        row = s_off[myle[j]] + grank;
    }
    if (row >= p.cap) row = -1;              // unreachable for a consistent histogram; keeps writes in bounds
    p.slot_row[t * k + j] = row;
    if (row >= 0) {
      p.row_token[row] = (int32_t)t;
      if (p.row_weight) p.row_weight[row] = p.topk_w[t * k + j];
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

int64_t permute_blocks(int64_t T) { return (T + CH - 1) / CH; }

hipError_t launch_permute(const PermuteProblem& p, hipStream_t stream, int (*between)()) {
  const int64_t nblk = permute_blocks(p.T);
  hipLaunchKernelGGL(k_chunk_count, dim3((unsigned)nblk), dim3(64), p.E_local * sizeof(int), stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_chunk_scan, dim3((unsigned)p.E_local), dim3(256), 0, stream, p, (int)nblk);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (between && between() != 0) return hipErrorUnknown;
  hipLaunchKernelGGL(k_rank, dim3((unsigned)nblk), dim3(64 * RW), (p.E_local + 1) * sizeof(int), stream, p);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (p.x_perm == nullptr) return hipSuccess;
  hipLaunchKernelGGL(k_gather, dim3((unsigned)((p.T + 3) / 4)), dim3(256), 0, stream, p);
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
