// Internal declarations shared by the kernel sources and the C-ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace moe {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

// Tile shape of the bf16 grouped GEMM: chosen from the rows per group, or
// the skinny 32x256 shape (used by the router GEMM, whose N is the expert
// count).
enum GemmTile : int { GEMM_TILE_AUTO = 0, GEMM_TILE_SKINNY = 1, GEMM_TILE_M64 = 2 };

// Epilogue of the grouped GEMM.
enum GemmEpilogue : int {
  EPI_STORE = 0,   // C = A·Bᵀ
  EPI_SWIGLU = 1,  // C = silu(A·B0ᵀ) * (A·B1ᵀ)
};

// One grouped GEMM "C[r] = op(A[gather[r]] · B_g)" over row segments.
//   A       : [*][K] row-major; row r of the problem reads A row gather[r]
//             (gather == nullptr: A row r).
//   offsets : [groups+1] device array; group g owns rows [offsets[g], offsets[g+1]).
//             nullptr: a single group of M rows.
//   B0, B1  : [groups][N][K] row-major (B1 only for EPI_SWIGLU).
//   C       : [M][ldc], N columns written per row.
// Malformed offsets or gather indices are clamped into range: they give
// unspecified results but never an out-of-bounds access.
struct GemmProblem {
  const void* A;
  int32_t a_rows;  // rows of A; gathered indices are clamped into [0, a_rows)
  const int32_t* gather;
  const int32_t* offsets;
  int32_t groups;
  int32_t M;  // upper bound on the rows (exact when offsets == nullptr)
  const void* B0;
  const void* B1;
  int32_t N;
  int32_t K;
  void* C;
  int32_t ldc;
  // K split (bf16 EPI_STORE with fp32 output only): split s sums the k-steps
  // [s*q, (s+1)*q), q = ceil(K/64 / ksplit), into C + s*c_split_stride.
  int32_t ksplit;
  int64_t c_split_stride;
  int32_t tile;  // GemmTile
  // Weight-streaming kernel only: one extra group (the shared expert, fused
  // into the routed launch) of x_rows rows of xA, taken in order (no gather),
  // with packed weights xB (one expert, same N and K) and output rows in xC
  // (leading dimension ldc). x_rows == 0: none.
  const void* xA;
  const void* xB;
  void* xC;
  int32_t x_rows;
  // Weight-streaming kernel only: 8 queue heads (one per XCD), zero at
  // launch, from which workgroups claim tiles after their first (nullptr:
  // a static round-robin schedule).
  int32_t* tile_queue;
  // Weight-streaming kernel, EPI_SWIGLU only: A holds int8 (or, with a_fp8,
  // E4M3) codes ([*][K] bytes) of rows whose fp32 scales are a_scale[A row]; every output row's
  // gate and up sums are multiplied by its row's scale before the SwiGLU.
  // The extra group must be empty (x_rows == 0). nullptr: A is bf16.
  const float* a_scale;
  // With a_scale: the codes are FP8 (OCP E4M3) values instead of int8.
  int32_t a_fp8;
  // Weight-streaming kernel only: group g owns rows [offsets[g], seg_end[g])
  // instead of [offsets[g], offsets[g+1]) (nullptr: adjacent segments), so a
  // call can cover part of every group's rows.
  const int32_t* seg_end;
  // 1: the groups' segments hold exactly M rows between them (a call over
  // every group of a dispatch), so M / groups is their average size; 0: M
  // only bounds them (a range of groups, or row segments).
  int32_t rows_exact;
  // Weight-streaming kernel only: at most this many workgroups (0: one per
  // compute unit), leaving compute units to kernels on other streams.
  int32_t max_wg;
  // Compute-bound kernel, EPI_STORE with offsets: workspace for splitting the
  // K range of the short remainder blocks (dense_part_bytes of it; nullptr:
  // no split). See dense_part_bytes().
  void* dense_part;
  int64_t dense_part_bytes;
  int32_t part_ks;  // set by the launcher: K parts of a remainder block (1: none)
  // Weight-streaming FFN launch (launch_ffn_stream) only: completion
  // counters, zero at launch: [g] counts the finished GEMM1 tiles of group g
  // (the extra group at [groups]); [groups + 1] is set when a GEMM2 tile gave
  // up waiting for its rows (never, unless tiles are lost); [groups + 2]
  // counts the workgroups done with GEMM1.
  int32_t* deps;
};

// Ints of the completion counters of a fused FFN launch: up to 256 groups,
// the extra group, the wait flag, the finished-workgroup count.
constexpr int kFfnDepsInts = 260;

// Workspace the compute-bound GEMM2 may use to split the K range of its
// short remainder blocks, for an FFN of `groups` groups over `rows` rows with
// output width n and reduction length k (0 when it never splits).
size_t dense_part_bytes(int64_t rows, int32_t groups, int32_t n, int32_t k);

// bf16 MFMA grouped GEMM (gfx950). out_f32 selects an fp32 output (EPI_STORE
// only); otherwise outputs are bf16.
hipError_t launch_gemm_bf16(const GemmProblem& p, int epilogue, bool out_f32, hipStream_t s);
// Weight-streaming bf16 grouped GEMM over packed weights (B0 = packed buffer;
// N % 128 == 0 for EPI_SWIGLU, N % 256 == 0 for EPI_STORE, K % 64 == 0).
hipError_t launch_gemm_stream(const GemmProblem& p, int epilogue, hipStream_t s);
// Compute-bound grouped GEMM over the same packed weights (gemm_dense.hip):
// 256x256 tiles with both operands shared through LDS, for groups of many
// rows (M exact, rows_exact, and an average >= 512 per group, at most 256
// groups), no extra group, no quantized tokens, no row segments, K % 128 == 0
// and K >= 256 (max_wg caps its grid too). launch_gemm_stream hands eligible
// problems to it.
bool gemm_dense_eligible(const GemmProblem& p);
hipError_t launch_gemm_dense(const GemmProblem& p, int epilogue, hipStream_t s);
// Zeroes n queue heads of launch_gemm_stream (a one-workgroup kernel, so
// it can be captured in a graph).
hipError_t launch_queue_reset(int32_t* q, int n, hipStream_t s);

// The whole weight-streaming expert FFN in one launch: every workgroup runs
// GEMM1 tiles (up: EPI_SWIGLU, bf16 tokens) until none is left, then GEMM2
// tiles (down: EPI_STORE), each of which first waits until every GEMM1 tile
// of its group has stored its rows of h. up.deps (== down.deps, zero at
// launch) holds the counters; up.tile_queue and down.tile_queue 8 zeroed
// heads each. Returns hipErrorNotSupported when the problem does not fit
// this launch (the caller then runs the two GEMMs as separate launches).
hipError_t launch_ffn_stream(const GemmProblem& up, const GemmProblem& down, hipStream_t s);
// Packs [E][N][K] row-major weights (gate_up: w0 = gate, w1 = up) into the
// streaming kernel's layout.
hipError_t launch_pack(const void* w0, const void* w1, void* dst, int E, int N, int K, bool gate_up, hipStream_t s);
// fp32 grouped GEMM (vector ALU), same semantics, fp32 in and out.
hipError_t launch_gemm_f32(const GemmProblem& p, int epilogue, hipStream_t s);

struct RouteParams {
  // logits = sum over s < nsplit of logits_in[s*split_stride + t*E + e],
  // summed in ascending s; written to logits_out when that is not null.
  const float* logits_in;
  int32_t nsplit;
  int64_t split_stride;
  float* logits_out;
  const float* bias;    // [E] or nullptr
  int32_t T, E, k, n_groups, topk_groups, score, renorm;
  float scale;
  int32_t* topk_idx;  // [T][k]
  float* topk_w;      // [T][k]
};
hipError_t launch_route(const RouteParams& p, hipStream_t s);

// Dispatch scratch: per 64-token chunk, an expert bitmask of the chunk's
// tokens ([chunks][E] uint64) and the rank base of the chunk inside every
// expert's segment ([chunks][E] int32).
constexpr int kDispatchChunk = 64;
struct DispatchParams {
  const int32_t* topk_idx;
  int32_t T, E, k;
  uint64_t* masks;
  int32_t* bases;
  int32_t* counts;
  int32_t* offsets;
  int32_t* sorted_token;
  int32_t* sorted_assign;  // may be nullptr
  int32_t* inv_perm;
  // Optional: n_zero ints at `zero` (the expert GEMMs' tile-queue heads) set
  // to 0 by the scan kernel, saving a launch before the expert FFN.
  int32_t* zero;
  int32_t n_zero;
};
hipError_t launch_dispatch(const DispatchParams& p, hipStream_t s);
// Library-owned dispatch scratch (moe_dispatch_noalloc): room for the masks
// and bases of ceil(T / kDispatchChunk) * E <= kDispatchNoAllocItems items
// (masks first, then the bases at byte kDispatchNoAllocItems * 8).
constexpr size_t kDispatchNoAllocItems = 262144;
constexpr size_t kDispatchNoAllocBytes = kDispatchNoAllocItems * (8 + 4);
// Device address of this device's copy of that scratch (looked up once per
// device with hipGetSymbolAddress, then cached; allocates nothing).
hipError_t dispatch_noalloc_scratch(void** out);

struct CombineParams {
  const void* y_perm;      // [T*k][d]
  const int32_t* inv_perm; // [T*k]
  const float* topk_w;     // [T][k]
  const void* shared_out;  // [T][d] or nullptr
  void* out;               // [T][d]
  int32_t T, k, d;
};
hipError_t launch_combine(const CombineParams& p, bool bf16, hipStream_t s);

// Per-token quantization. int8: codes[t][c] = rne(x[t][c] / scale[t])
// clamped to +-127, scale[t] = max_c |x[t][c]| / 127; fp8: E4M3 codes of
// x[t][c] / scale[t] (clamped to +-448, round to nearest even), scale[t] =
// max_c |x[t][c]| / 448. A zero row: scale 0, codes 0. x bf16 [T][d],
// d % 64 == 0; codes [T][d] bytes; scales fp32 [T].
hipError_t launch_quantize(const void* x, int8_t* codes, float* scales, int T, int d, bool fp8, hipStream_t s);

// Receive side of expert parallelism: fills the self (mode 0) or remote
// (mode 1) rows of experts [e0, e1) of a receive buffer whose expert e owns
// rows [offsets[e], offsets[e+1]), self rows below self_end[e]:
// dst[r] = src[row_token[r]] (rows of row_bytes bytes, a multiple of 16).
// Indices are clamped into range. max_wg > 0 limits the workgroups.
struct EpCopyParams {
  const void* src;  // [src_rows][row_bytes]
  int32_t src_rows;
  const int32_t* row_token;  // [n_rows]
  const int32_t* offsets;    // [E+1]
  const int32_t* self_end;   // [E]
  int32_t e0, e1, mode, n_rows, row_bytes;
  void* dst;  // [n_rows][row_bytes]
};
hipError_t launch_ep_copy(const EpCopyParams& p, int max_wg, hipStream_t s);
// Receive-buffer layout of local experts [e_first, e_first + e_count) from
// this GPU's and the peer's dispatch (offsets over the global experts and
// the expert-sorted token lists): offsets [e_count+1], self_end [e_count],
// row_token [capacity] (rows past the capacity are not written).
struct EpPlanParams {
  const int32_t* self_offsets;
  const int32_t* self_sorted;
  int32_t self_total;
  const int32_t* peer_offsets;
  const int32_t* peer_sorted;
  int32_t peer_total;
  int32_t e_first, e_count, capacity;
  int32_t* row_token;
  int32_t* offsets;
  int32_t* self_end;
};
hipError_t launch_ep_plan(const EpPlanParams& p, hipStream_t s);

// Number of compute units of the current device (cached per device).
int device_cu_count();
// Raises kernel `kern`'s dynamic LDS limit to `bytes` on the current device,
// once per (kernel, device): the attribute belongs to the device's copy of the
// kernel. Later calls return the first call's status.
hipError_t set_dynamic_lds(const void* kern, int bytes);

}  // namespace moe
