// Grouped GEMM on gfx950 bf16 MFMA (v_mfma_f32_32x32x16_bf16), fp32 accumulation.
//
// One launch serves every group (local expert) of a batch: the row segment of group g
// is [offsets[g], offsets[g+1]) -- the monotone [E+1] row-offset array of the paper's
// kernel-generation section -- read from device memory, so the number of rows never
// travels to the host.  Each workgroup builds the tile table of the launch in LDS
// (ceil(m_g / BM) x n-tiles per group, a block-wide prefix sum) and then walks tiles
// persistently.  Tiles of one group are ordered m-fastest so that the tiles sharing a
// weight tile are adjacent, and adjacent tiles are handed to workgroups of the same
// XCD (workgroup i runs on XCD i mod 8), so a weight tile is fetched from HBM once per
// XCD L2 rather than once per m-tile.
//
// Operand roles: the weight tile is the MFMA A operand (rows = output features) and the
// token tile the B operand (columns = tokens), so each lane ends with 4 consecutive
// output features of one token: 8-byte bf16 stores along the output row.
//
// LDS: both tiles are [rows][64] bf16 (128 B per row = 8 chunks of 16 B); chunk c of row r
// lives at chunk c ^ ((r >> 1) & 7), so the 16 lanes of one ds_read_b128 phase (16
// consecutive rows, one logical chunk) cover all 64 banks once.  Two stages: while the
// MFMAs consume stage s, the next K slice is already in registers and is written to
// stage s^1 afterwards (one barrier per K slice).
#include "common.hpp"
#include "kernels.hpp"

namespace moe {
namespace {

constexpr int BK = 64;
constexpr int NT = 256;

__device__ __forceinline__ int swz(int row, int chunk) { return row * BK + ((chunk ^ ((row >> 1) & 7)) << 3); }

__device__ __forceinline__ bf16x8 lds_frag(const bf16_t* tile, int row, int chunk) {
  return *reinterpret_cast<const bf16x8*>(tile + swz(row, chunk));
}

// Block-wide exclusive scan of one int per thread (NT threads); returns the block total.
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
  for (int w = 0; w < NT / 64; ++w) {
    int t = s_tmp[w];
    if (w < wave) wbase += t;
    total += t;
  }
  excl = wbase + inc - v;
  __syncthreads();
  return total;
}

template <int BM, int BN, int EPI>
__global__ __launch_bounds__(NT) void k_grouped_gemm(GemmProblem p) {
  constexpr int WM = BM / 2, WN = BN / 2;      // 2 x 2 waves
  constexpr int FM = WM / 32, FN = WN / 32;    // 32x32 fragments per wave
  constexpr int XCH = BM * 8 / NT, WCH = BN * 8 / NT;
  constexpr int OUTN = (EPI == EPI_SWIGLU) ? BN / 2 : BN;
  static_assert(FM >= 1 && FN >= 1 && XCH >= 1 && WCH >= 1, "tile too small");
  static_assert(EPI != EPI_SWIGLU || FN % 2 == 0, "SwiGLU pairs gate and up fragments");

  extern __shared__ __align__(16) uint8_t smem[];
  bf16_t* sX = reinterpret_cast<bf16_t*>(smem);              // [2][BM][BK]
  bf16_t* sW = sX + 2 * BM * BK;                              // [2][BN][BK]
  __shared__ int s_off[kMaxGroups + 1];
  __shared__ int s_tp[kMaxGroups + 1];
  __shared__ int s_tmp[NT / 64];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int tiles_n = (p.N + OUTN - 1) / OUTN;

  // ---- tile table: s_tp[g] = first tile of group g ----
  int groups = p.groups;
  if (p.offsets) {
    // clamp to [0, max_rows]: any offsets content keeps every access inside the buffers
    const int cap = (int)p.max_rows;
    for (int g = tid; g <= groups; g += NT) s_off[g] = min(max(p.offsets[g], 0), cap);
  } else {
    groups = 1;
    if (tid == 0) { s_off[0] = 0; s_off[1] = (int)p.rows_single; }
  }
  __syncthreads();
  constexpr int PER = (kMaxGroups + NT - 1) / NT;
  int loc[PER];
  int lsum = 0;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    int g = tid * PER + i;
    int m = g < groups ? max(s_off[g + 1] - s_off[g], 0) : 0;
    loc[i] = ((m + BM - 1) / BM) * tiles_n;
    lsum += loc[i];
  }
  int excl;
  const int total = block_exclusive_scan(lsum, s_tmp, excl);
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    int g = tid * PER + i;
    if (g < groups) s_tp[g] = excl;
    excl += loc[i];
  }
  if (tid == 0) s_tp[groups] = total;
  __syncthreads();

  const int G = gridDim.x;
  const int slot = (G % 8 == 0) ? (int)(blockIdx.x % 8) * (G / 8) + (int)(blockIdx.x / 8) : (int)blockIdx.x;

  for (int base = 0; base < total; base += G) {
    const int tile = base + slot;
    if (tile >= total) break;
    // group of this tile: last g with s_tp[g] <= tile
    int lo = 0, hi = groups;             // s_tp[groups] == total > tile
    while (hi - lo > 1) {
      int mid = (lo + hi) >> 1;
      if (s_tp[mid] <= tile) lo = mid; else hi = mid;
    }
    const int g = lo;
    const int row0g = s_off[g], row_end = s_off[g + 1];
    const int mt = (row_end - row0g + BM - 1) / BM;
    const int local = tile - s_tp[g];
    const int mi = local % mt, ni = local / mt;
    const int row0 = row0g + mi * BM;
    const bf16_t* Wg = p.W + (int64_t)g * p.w_group_stride;

    // ---- per-thread global chunk pointers ----
    const bf16_t* xp[XCH];
    int xs[XCH];
#pragma unroll
    for (int i = 0; i < XCH; ++i) {
      int c = tid + i * NT, r = c >> 3, ch = c & 7;
      int row = min(row0 + r, row_end - 1);
      xp[i] = p.X + (int64_t)row * p.ldx + ch * 8;
      xs[i] = swz(r, ch);
    }
    const bf16_t* wp[WCH];
    int ws[WCH];
#pragma unroll
    for (int i = 0; i < WCH; ++i) {
      int c = tid + i * NT, r = c >> 3, ch = c & 7;
      int wrow;
      if (EPI == EPI_SWIGLU) {
        int half = r >= BN / 2;
        int f = min(ni * (BN / 2) + (r - half * (BN / 2)), p.N - 1);
        wrow = f + half * p.N;
      } else {
        wrow = min(ni * BN + r, p.N - 1);
      }
      wp[i] = Wg + (int64_t)wrow * p.K + ch * 8;
      ws[i] = swz(r, ch);
    }

    const int nk = (p.K + BK - 1) / BK;
    u32x4 rx[XCH], rw[WCH];
    auto gload = [&](int kt) {
      const int k0 = kt * BK;
#pragma unroll
      for (int i = 0; i < XCH; ++i) {
        int ch = (tid + i * NT) & 7;
        rx[i] = (k0 + ch * 8 < p.K) ? ld16(xp[i] + k0) : u32x4{0, 0, 0, 0};
      }
#pragma unroll
      for (int i = 0; i < WCH; ++i) {
        int ch = (tid + i * NT) & 7;
        rw[i] = (k0 + ch * 8 < p.K) ? ld16(wp[i] + k0) : u32x4{0, 0, 0, 0};
      }
    };
    auto lstore = [&](int st) {
      bf16_t* dX = sX + st * BM * BK;
      bf16_t* dW = sW + st * BN * BK;
#pragma unroll
      for (int i = 0; i < XCH; ++i) st16(dX + xs[i], rx[i]);
#pragma unroll
      for (int i = 0; i < WCH; ++i) st16(dW + ws[i], rw[i]);
    };

    f32x16 acc[FM][FN];
#pragma unroll
    for (int a = 0; a < FM; ++a)
#pragma unroll
      for (int b = 0; b < FN; ++b)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[a][b][q] = 0.f;

    // weight-row base of each fragment of this wave
    int wbase[FN];
#pragma unroll
    for (int b = 0; b < FN; ++b) {
      if (EPI == EPI_SWIGLU)
        wbase[b] = (b < FN / 2) ? wn * (BN / 4) + b * 32 : BN / 2 + wn * (BN / 4) + (b - FN / 2) * 32;
      else
        wbase[b] = wn * WN + b * 32;
    }

    __syncthreads();            // previous tile's last LDS reads are done
    gload(0);
    lstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      const int st = kt & 1;
      if (kt + 1 < nk) gload(kt + 1);
      const bf16_t* cX = sX + st * BM * BK;
      const bf16_t* cW = sW + st * BN * BK;
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        const int ch = ks * 2 + (lane >> 5);
        bf16x8 fw[FN], fx[FM];
#pragma unroll
        for (int b = 0; b < FN; ++b) fw[b] = lds_frag(cW, wbase[b] + (lane & 31), ch);
#pragma unroll
        for (int a = 0; a < FM; ++a) fx[a] = lds_frag(cX, wm * WM + a * 32 + (lane & 31), ch);
#pragma unroll
        for (int a = 0; a < FM; ++a)
#pragma unroll
          for (int b = 0; b < FN; ++b)
            acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[b], fx[a], acc[a][b], 0, 0, 0);
      }
      if (kt + 1 < nk) lstore(st ^ 1);
      __syncthreads();
    }

    // ---- epilogue: lane holds token column (lane & 31); features 8q + 4(lane>>5) + 0..3 ----
#pragma unroll
    for (int a = 0; a < FM; ++a) {
      const int row = row0 + wm * WM + a * 32 + (lane & 31);
      if (row >= row_end) continue;
      if (EPI == EPI_SWIGLU) {
        bf16_t* yrow = reinterpret_cast<bf16_t*>(p.Y) + (int64_t)row * p.ldy;
#pragma unroll
        for (int b = 0; b < FN / 2; ++b) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int col = ni * (BN / 2) + wn * (BN / 4) + b * 32 + 8 * q + 4 * (lane >> 5);
            if (col >= p.N) continue;
            float o[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              float gt = acc[a][b][4 * q + e], up = acc[a][b + FN / 2][4 * q + e];
              o[e] = gt / (1.0f + __expf(-gt)) * up;
            }
            uint2 v;
            v.x = pack_bf16x2(o[0], o[1]);
            v.y = pack_bf16x2(o[2], o[3]);
            *reinterpret_cast<uint2*>(yrow + col) = v;
          }
        }
      } else if (EPI == EPI_BF16) {
        bf16_t* yrow = reinterpret_cast<bf16_t*>(p.Y) + (int64_t)row * p.ldy;
#pragma unroll
        for (int b = 0; b < FN; ++b) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int col = ni * BN + wn * WN + b * 32 + 8 * q + 4 * (lane >> 5);
            if (col >= p.N) continue;
            uint2 v;
            v.x = pack_bf16x2(acc[a][b][4 * q + 0], acc[a][b][4 * q + 1]);
            v.y = pack_bf16x2(acc[a][b][4 * q + 2], acc[a][b][4 * q + 3]);
            *reinterpret_cast<uint2*>(yrow + col) = v;
          }
        }
      } else {
        float* yrow = reinterpret_cast<float*>(p.Y) + (int64_t)row * p.ldy;
#pragma unroll
        for (int b = 0; b < FN; ++b) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int col = ni * BN + wn * WN + b * 32 + 8 * q + 4 * (lane >> 5);
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (col + e < p.N) yrow[col + e] = acc[a][b][4 * q + e];
          }
        }
      }
    }
  }
}

struct DevInfo {
  int cus = 0;
  int lds = 0;
};
DevInfo g_dev[64];

DevInfo& dev_info() {
  static DevInfo fallback{256, 65536};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return fallback;
  DevInfo& d = g_dev[dev];
  if (d.cus == 0) {
    int n = 0, l = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    if (hipDeviceGetAttribute(&l, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess || l <= 0)
      l = 65536;
    d.lds = l;
    d.cus = n;
  }
  return d;
}
int cu_count() { return dev_info().cus; }
int lds_limit() { return dev_info().lds; }

template <int BM, int BN, int EPI>
hipError_t launch_tile(const GemmProblem& p, hipStream_t stream) {
  constexpr int OUTN = (EPI == EPI_SWIGLU) ? BN / 2 : BN;
  const size_t lds = (size_t)2 * (BM + BN) * BK * sizeof(bf16_t);
  if (lds + 2 * (kMaxGroups + 1) * sizeof(int) + 64 > (size_t)lds_limit()) return hipErrorInvalidConfiguration;
  static bool attr_set = false;   // idempotent attribute, racing writers store the same value
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_grouped_gemm<BM, BN, EPI>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const int64_t tiles_n = (p.N + OUTN - 1) / OUTN;
  const int64_t groups = p.offsets ? p.groups : 1;
  const int64_t rows = p.offsets ? p.max_rows : p.rows_single;
  const int64_t upper = tiles_n * ((rows + BM - 1) / BM + groups);
  const int64_t resident = (int64_t)cu_count() * 2;
  int64_t grid = upper < resident ? upper : resident;
  if (grid >= 8) grid -= grid % 8;
  if (grid < 1) grid = 1;
  hipLaunchKernelGGL((k_grouped_gemm<BM, BN, EPI>), dim3((unsigned)grid), dim3(NT), lds, stream, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_grouped_gemm(const GemmProblem& p, hipStream_t stream) {
  switch (p.epi) {
    case EPI_SWIGLU: return launch_tile<128, 128, EPI_SWIGLU>(p, stream);
    case EPI_BF16: return launch_tile<128, 128, EPI_BF16>(p, stream);
    case EPI_F32: return launch_tile<64, 64, EPI_F32>(p, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace moe
