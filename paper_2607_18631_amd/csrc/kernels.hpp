// Host-side launchers of the gfx950 kernels (internal to libmoe_mi355x.so), and the host-only
// size arithmetic of their workspaces (sizes.cpp).
#pragma once
#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include <mutex>

namespace moe {

typedef uint16_t bf16_t;

constexpr int kMaxGroups = 1024;  // E_local limit of the grouped GEMM's in-LDS tile table

enum Epilogue { EPI_BF16 = 0, EPI_SWIGLU = 1, EPI_F32 = 2, EPI_SCATTER = 3, EPI_SWIGLU_BWD = 4 };

// One grouped GEMM  Y[r, n] = sum_k X[r, k] * W_g[n, k]  for every group g and every
// row r in [offsets[g], offsets[g+1]).  Both operands are K-contiguous.
// EPI_SWIGLU: W_g holds 2N rows (gate rows [0,N), up rows [N,2N)) and
//             Y[r, n] = bf16(silu(gate) * up).
// EPI_SWIGLU_BWD: the up-projection recomputed in the backward; with gate h and up u of row r,
//             feature n, and dA = dact[r, n]:  Y[r, n] = bf16(dA * u * silu'(h)),
//             Y[r, N + n] = bf16(dA * silu(h)) (row stride ldy = 2N), and act_out[r, n] =
//             bf16(silu(h) * u) (row stride N), the activation the weight gradient of W2 needs.
// EPI_SCATTER: float32 Y rows are token rows: Y[tok(r), n] += w(r) * (X W_g^T)[r, n] by
//             atomics, tok(r) = scatter_token[r] and w(r) = scatter_weight[r] for the grouped
//             rows (identity and 1 when the pointers are null, and for the extra group).
struct GemmProblem {
  const bf16_t* X;            // token rows, row stride ldx (elements)
  int64_t ldx;
  const int32_t* offsets;     // device [groups+1]; nullptr = one group of rows_single rows;
                              // with seg_stride > 0: device [groups] row counts
  int32_t groups;
  int64_t rows_single;
  int64_t max_rows;           // host-known bound of offsets[groups] (grid sizing only)
  const bf16_t* W;            // weights of group 0, row stride K
  int64_t w_group_stride;     // elements between consecutive groups' weights
  int32_t N;                  // output columns
  int32_t K;
  void* Y;                    // bf16 or f32 output, row stride ldy (elements)
  int64_t ldy;
  int32_t epi;
  // optional extra group on its own operands (the shared expert run inside the routed launch):
  // rows [0, rows2) of X2 against W2 into Y2, same N, K, ldx and ldy; rows2 = 0 means none
  const bf16_t* X2;
  const bf16_t* W2;
  void* Y2;
  int32_t rows2;
  int32_t rows2_tile;         // m-tile height of the extra group: 0 = the launch's, else a multiple
                              // of 32 below it (its tiles then run with dead blocks)
  // K split (EPI_F32, one group, no extra group): ksplit > 1 runs the K range in ksplit
  // chunks, chunk c writing its fp32 partial product at Y + c * y_split_stride
  int32_t ksplit;
  int64_t y_split_stride;
  // gathered rows (the permutation folded into the copies): when row_index is set, row r of
  // the grouped part is row row_index[r] of X (X has x_rows rows; indices are clamped to them)
  const int32_t* row_index;
  int64_t x_rows;
  // expected rows per group (0 = unknown): selects the tile shape (the row counts themselves
  // stay on the device)
  int64_t rows_hint;
  // equal-stride segments (masked-decode layout): group g owns rows
  // [g * seg_stride, g * seg_stride + min(offsets[g], seg_stride)); 0 = monotone offsets
  int32_t seg_stride;
  // EPI_SCATTER: token and gate of every grouped row; tokens outside [0, scatter_rows) are skipped
  const int32_t* scatter_token;
  const float* scatter_weight;
  int64_t scatter_rows;
  // EPI_SWIGLU_BWD: gradient of the activation [rows, N] and the recomputed activation
  const bf16_t* dact;
  bf16_t* act_out;
};

hipError_t launch_grouped_gemm(const GemmProblem& p, hipStream_t stream);

// compute units and the LDS bytes per workgroup of the current device (queried once per device)
int cu_count();
int lds_limit();

// Resident workgroups per CU of one kernel, per device: the first launch on a device raises the
// kernel's dynamic-LDS limit to `lds` and queries the occupancy, once (std::call_once); later
// launches read the stored result.  Returns 0 and sets err on failure.
constexpr int kMaxDevices = 64;
struct OccCache {
  std::once_flag once[kMaxDevices];
  int per_cu[kMaxDevices] = {};
  hipError_t err[kMaxDevices] = {};
};
int kernel_occupancy(OccCache& c, const void* fn, int nth, size_t lds, hipError_t& err);

// Grouped GEMMs of the expert-MLP backward:  Y[m, n] = sum_k X[m, k] * W[n, k]  with each
// operand either K-major (element (r, k) at base + r * ld + k) or MN-major (element (k, r) at
// base + k * ld + r, the transposed layout of a row-major activation or weight).
//  mode BWD_ROWS: group g owns rows [seg_begin(g), seg_end(g)) of X and Y (as the forward),
//                 K = p.K, weights W + g * w_group_stride;
//  mode BWD_KSEG: group g reduces over the rows [seg_begin(g), seg_end(g)) of two row-major
//                 activations (X and W both MN-major, k = row): Y_g = Y + g * y_group_stride,
//                 an M x N matrix per group (weight gradients; an empty group writes zeros).
// Segments: monotone offsets[groups + 1], or seg_stride > 0 with offsets = counts[groups]
// (group g owns [g * seg_stride, g * seg_stride + min(count, seg_stride))).
enum BwdMode { BWD_ROWS = 0, BWD_KSEG = 1 };
struct GemmBwdProblem {
  int32_t mode;
  bool x_mn, w_mn;            // operand layouts (MN-major when set)
  const bf16_t* X;
  int64_t ldx;
  const bf16_t* W;
  int64_t ldw;
  int64_t w_group_stride;     // BWD_ROWS
  const int32_t* offsets;
  int32_t groups;
  int32_t seg_stride;
  int64_t max_rows;           // host-known bound of the rows (grid sizing, offsets clamp)
  int64_t rows_hint;          // expected rows per group (BWD_ROWS tile shape), 0 = unknown
  int32_t M;                  // BWD_KSEG: output rows per group
  int32_t N;                  // output columns
  int32_t K;                  // BWD_ROWS: reduction length
  bf16_t* Y;
  int64_t ldy;
  int64_t y_group_stride;     // BWD_KSEG
  float* Yf;                  // BWD_KSEG: when set, float32 results here (same strides) instead of Y
};
hipError_t launch_gemm_bwd(const GemmBwdProblem& p, hipStream_t stream);

// (BM, BN, BK) of the tile the fp32-output GEMM (router logits) runs with: the 256 x 256 tile
// (K-split for parallelism) when there are many tokens and experts, else 64 x 64 tiles
struct TileShape {
  int bm, bn, bk;
};
TileShape f32_tile(int64_t rows, int n);

// Number of K chunks the router-logits GEMM (T x E outputs, K = d) runs in: enough (m, n, k)
// tiles for one per compute unit of the chip, every chunk non-empty.  Depends on the shape
// only, so workspace sizes do not depend on the device.
int logits_splits(int64_t T, int E, int K);

struct GateProblem {
  const float* logits;        // nsplit partial sums, each [T, E]: logits = sum of the partials
  int32_t nsplit;
  int64_t split_stride;       // elements between partials
  const float* bias;          // [E] or nullptr
  int64_t T;
  int32_t E, top_k, gate, n_group, topk_group, renormalize;
  int32_t group_size;         // E / n_group
  float routed_scale;
  int32_t* topk_idx;          // [T, top_k]
  float* topk_w;              // [T, top_k]
  float* keys_out;            // [T, E] or nullptr
};
hipError_t launch_gate(const GateProblem& p, hipStream_t stream);

struct PermuteProblem {
  const int32_t* topk_idx;    // [T, top_k]
  const bf16_t* x;            // [T, d]
  int64_t T;
  int32_t d, top_k, e_begin, E_local;
  int32_t* counts;            // [E_local]
  int32_t* offsets;           // [E_local + 1]
  int32_t* row_token;         // [cap]
  int32_t* slot_row;          // [T, top_k]
  bf16_t* x_perm;             // [cap, d]; nullptr: no row copy (the GEMM gathers the rows itself)
  int64_t cap;                // rows of row_token / x_perm
  int32_t expert_capacity;    // > 0: masked-decode layout (rows e * C + rank, rank < C)
  const float* topk_w;        // [T, top_k]; read only when row_weight is set
  float* row_weight;          // [cap] gate of each row, or nullptr
  int32_t* super_count;       // workspace [nsuper, E_local]: local slots per 512-token super-chunk
  int32_t* super_base;        // workspace [nsuper, E_local]: their exclusive scan (wide tables only)
  int32_t* totals;            // workspace [E_local]: expert totals (wide tables only)
  uint64_t* chunk_mask;       // workspace [nsuper * 8, E_local]: per 64-token chunk, lanes holding each expert
  int32_t* chunk_base;        // workspace [nsuper * 8, E_local]: the chunk's base inside its super-chunk
};
// Permutation geometry: 64-token chunks (one wave), kPermSuper chunks per super-chunk.
constexpr int kPermChunk = 64;
constexpr int kPermSuper = 8;
// super-chunks of T tokens, and the permutation workspace: byte offsets of its arrays and size
int64_t permute_supers(int64_t T);
struct PermuteWs {
  size_t super_count, super_base, totals, chunk_mask, chunk_base, bytes;
};
PermuteWs permute_ws(int64_t T, int E_local);
// `between` (may be empty) runs on the host after the histogram launches and before the
// permute launch (used to record a timing event between the two steps).
hipError_t launch_permute(const PermuteProblem& p, hipStream_t stream, int (*between)() = nullptr);

struct CombineProblem {
  const bf16_t* y_perm;       // [cap, d]
  const int32_t* slot_row;    // [T, top_k]
  const float* topk_w;        // [T, top_k]
  const bf16_t* shared_y;     // [T, d] or nullptr
  bf16_t* out;                // [T, d]
  int64_t T;
  int64_t cap;                // rows of y_perm; slot rows outside [0, cap) are skipped
  int32_t d, top_k;
};
hipError_t launch_combine(const CombineProblem& p, hipStream_t stream);

// Scratch of moe_permute_noalloc: a device array of this many bytes owned by the library (one
// per device, shared by every call on it).  permute_scratch returns its device address on the
// current device (looked up once per device).
constexpr size_t kPermuteScratchBytes = size_t(1) << 20;
hipError_t permute_scratch(void** ptr);

// The row copy of the permutation alone: x_perm[slot_row[t, j]] = x[t] for every local slot.
hipError_t launch_gather(const PermuteProblem& p, hipStream_t stream);

// ---- layer backward (around the expert-MLP backward GEMMs) ----
// dgate[t, j] = <dout[t], y_perm[slot_row[t, j]]> (0 for a slot without a local row) and
// dy_perm[slot_row[t, j]] = bf16(topk_w[t, j] * dout[t]).
struct CombineBwdProblem {
  const bf16_t* dout;         // [T, d]
  const bf16_t* y_perm;       // [cap, d]
  const int32_t* slot_row;    // [T, top_k]
  const float* topk_w;        // [T, top_k]
  float* dgate;               // [T, top_k]
  bf16_t* dy_perm;            // [cap, d]
  int64_t T, cap;
  int32_t d, top_k;
};
hipError_t launch_combine_bwd(const CombineBwdProblem& p, hipStream_t stream);

// dlogits [T, E] = d loss / d router logit (bf16), from the gate gradients and the forward's
// float32 keys recomputed from its logit partials; also writes seg = {0, T}.
struct GateBwdProblem {
  const float* logits;        // nsplit partials [T, E] of the forward's router GEMM
  int32_t nsplit;
  int64_t split_stride;
  const float* bias;          // [E] or nullptr (softmax keys)
  const int32_t* topk_idx;    // [T, top_k]
  const float* dgate;         // [T, top_k]
  int64_t T;
  int32_t E, top_k, gate, renormalize;
  float routed_scale;
  bf16_t* dlogits;            // [T, E]
  int32_t* seg;               // [2] or nullptr: {0, T}
  int32_t* segk;              // [nsegk + 1] or nullptr: {0, c, 2c, ..., T} (token chunks of segk_rows)
  int32_t nsegk;
  int64_t segk_rows;
};
hipError_t launch_gate_bwd(const GateBwdProblem& p, hipStream_t stream);

// out[t] = bf16( sum of rows[slot_row[t, j]] over the local slots (slot order) + extra0[t] + extra1[t] )
struct UnpermuteSumProblem {
  const bf16_t* rows;         // [cap, d]
  const int32_t* slot_row;    // [T, top_k]
  const bf16_t* extra0;       // [T, d] or nullptr
  const bf16_t* extra1;       // [T, d] or nullptr
  bf16_t* out;                // [T, d]
  int64_t T, cap;
  int32_t d, top_k;
};
hipError_t launch_unpermute_sum(const UnpermuteSumProblem& p, hipStream_t stream);

// out[i] = bf16( sum over s = 0 .. nparts-1, in that order, of parts[s * n + i] ), n % 4 == 0
hipError_t launch_sum_partials(const float* parts, int nparts, int64_t n, bf16_t* out, hipStream_t stream);

// acc[0 .. n) = 0 (a fill kernel, so the call can sit inside a captured graph); n % 4 == 0
hipError_t launch_zero_f32(float* acc, int64_t n, hipStream_t stream);
// out[i] = bf16(acc[i]) for i < n, n % 8 == 0
hipError_t launch_round_bf16(const float* acc, bf16_t* out, int64_t n, hipStream_t stream);

}  // namespace moe
