// Grouped bf16 GEMM on the gfx950 matrix cores (v_mfma_f32_32x32x16_bf16).
//
// This is the expert FFN of the MoE layer (App. M step 3; App. F GEMM1 +
// SwiGLU + GEMM2): every expert multiplies its segment of dispatched token
// rows by its own weight matrix. One kernel covers
//   * GEMM1 with the SwiGLU epilogue: h = silu(X·Wgᵀ) * (X·Wuᵀ), the gate and
//     up columns of one output column sitting in the same lane and register,
//   * GEMM2 and the router GEMM: C = X·Wᵀ (bf16 or fp32 output),
// with the token gather (row r reads x[sorted_token[r]]) fused into the
// A-tile load, so the permuted activations are never materialised.
//
// Structure
//   * Persistent grid: each workgroup walks tiles tile = vb, vb+G, ...; the
//     tile list (expert, m-tile, n-tile) is derived in the prologue from the
//     expert offsets, so no host round trip is needed and empty experts cost
//     nothing. vb is the XCD-aware virtual block id: workgroups are handed to
//     the 8 XCDs round-robin, so vb = (b % 8) * (G/8) + b/8 gives every XCD a
//     contiguous run of tiles, i.e. the tiles of one expert share that XCD's
//     L2 (A rows are re-read by every n-tile, B columns by every m-tile).
//   * Within an expert, tiles are ordered in groups of kGroupM m-tiles per
//     n-tile so that m-tiles sharing a B slice run side by side.
//   * K is walked in steps of 64 (128 bytes per row): global loads for step
//     s+1 are issued into registers before the MFMAs of step s, then stored to
//     the other half of a double-buffered LDS tile; one barrier per step.
//   * LDS rows are 128 bytes; the 16-byte chunk c of row r is stored at chunk
//     c ^ (r & 7), which makes both the row-wise stores and the column-wise
//     fragment reads (8 rows, same chunk) bank-conflict free.
//   * 4 waves per workgroup in a WGM x WGN grid; a wave owns FM x FN
//     32x32 accumulators. Fragments whose 32 rows all lie past the segment's
//     end are skipped (wave-uniform), so short expert segments do not pay for
//     the padding.
#include "moe_internal.h"

#include <mutex>
#include <type_traits>

namespace moe {
namespace {

constexpr int kThreads = 256;
constexpr int kGroupM = 4;

__device__ __forceinline__ int lds_off(int row, int chunk) {
  return (row << 7) + ((chunk ^ (row & 7)) << 4);
}

__device__ __forceinline__ float silu_f(float g) { return g / (1.0f + __expf(-g)); }

__device__ __forceinline__ void store_out(__bf16* C, size_t i, float v) { C[i] = static_cast<__bf16>(v); }
__device__ __forceinline__ void store_out(float* C, size_t i, float v) { C[i] = v; }

// Exclusive scan of one int per thread over a 256-thread block; returns the
// exclusive prefix and writes the block total to *total.
__device__ int block_exclusive_scan(int v, int* scratch /*[4]*/, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int n = __shfl_up(inc, o, 64);
    if (lane >= o) inc += n;
  }
  if (lane == 63) scratch[wave] = inc;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    int s = scratch[w];
    if (w < wave) base += s;
    tot += s;
  }
  *total = tot;
  return base + inc - v;
}

template <int BM, int BN, int WGM, int WGN, int EPI, bool OUT_F32>
__global__ void __launch_bounds__(kThreads)
gemm_bf16_kernel(GemmProblem p) {
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int FM = WTM / 32, FN = WTN / 32;
  constexpr int A_CH = BM / 32, B_CH = BN / 32;  // 16-byte chunks per thread per step
  static_assert(WGM * WGN == 4, "4 waves");
  static_assert(FM >= 1 && FN >= 1 && WTM % 32 == 0 && WTN % 32 == 0, "32x32 fragments");
  static_assert(EPI != EPI_SWIGLU || (FN % 2 == 0), "swiglu pairs gate/up fragments");
  using OutT = typename std::conditional<OUT_F32, float, __bf16>::type;

  extern __shared__ __attribute__((aligned(16))) char smem[];
  char* const As = smem;                 // [2][BM rows x 128 B]
  char* const Bs = smem + 2 * BM * 128;  // [2][BN rows x 128 B]
  __shared__ int tstart[257];
  __shared__ int scan_scratch[4];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int groups = p.offsets ? p.groups : 1;

  // ---- tile plan: m-tiles before every group -------------------------------
  {
    int mt = 0;
    if (tid < groups) {
      int c = p.M;
      if (p.offsets) {
        const int lo = min(max(p.offsets[tid], 0), p.M);
        c = min(max(p.offsets[tid + 1], lo), p.M) - lo;
      }
      mt = (c + BM - 1) / BM;
    }
    int total;
    const int ex = block_exclusive_scan(mt, scan_scratch, &total);
    if (tid < groups) tstart[tid] = ex;
    if (tid == 0) tstart[groups] = total;
    __syncthreads();
  }
  const int ncols_tile = (EPI == EPI_SWIGLU) ? BN / 2 : BN;
  const int Nt = (p.N + ncols_tile - 1) / ncols_tile;
  const int total_tiles = tstart[groups] * Nt;

  const int G = gridDim.x;
  const int b = blockIdx.x;
  const int vb = (G % 8 == 0) ? (b % 8) * (G / 8) + (b / 8) : b;

  const __bf16* const A = static_cast<const __bf16*>(p.A);
  const size_t K = (size_t)p.K;
  const int nk = p.K / 64;

  for (int tile = vb; tile < total_tiles; tile += G) {
    // ---- decode the tile --------------------------------------------------
    const int q = tile / Nt;
    int lo = 0, hi = groups - 1;  // largest e with tstart[e] <= q
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (tstart[mid] <= q) lo = mid; else hi = mid - 1;
    }
    const int e = lo;
    const int local = tile - tstart[e] * Nt;
    const int mte = tstart[e + 1] - tstart[e];
    const int grp = local / (kGroupM * Nt);
    const int first = grp * kGroupM;
    const int gsz = min(kGroupM, mte - first);
    const int within = local - grp * kGroupM * Nt;
    const int mloc = first + within % gsz;
    const int nt = within / gsz;
    const int gbeg = p.offsets ? min(max(p.offsets[e], 0), p.M) : 0;
    const int gend = p.offsets ? min(max(p.offsets[e + 1], gbeg), p.M) : p.M;
    const int row0 = gbeg + mloc * BM;
    const int rows = min(BM, gend - row0);
    const int n0 = nt * ncols_tile;

    // ---- per-thread global source pointers ------------------------------
    const int cchunk = tid & 7;
    const int rbase = tid >> 3;
    const __bf16* a_src[A_CH];
#pragma unroll
    for (int i = 0; i < A_CH; ++i) {
      const int r = rbase + 32 * i;
      if (r < rows) {
        const int ar = p.gather ? min(max(p.gather[row0 + r], 0), p.a_rows - 1) : row0 + r;
        a_src[i] = A + (size_t)ar * K + cchunk * 8;
      } else {
        a_src[i] = nullptr;
      }
    }
    const __bf16* b_src[B_CH];
    {
      const size_t gstride = (size_t)p.N * K;
      const __bf16* B0 = static_cast<const __bf16*>(p.B0) + (size_t)e * gstride;
      const __bf16* B1 = (EPI == EPI_SWIGLU) ? static_cast<const __bf16*>(p.B1) + (size_t)e * gstride : nullptr;
#pragma unroll
      for (int i = 0; i < B_CH; ++i) {
        const int r = rbase + 32 * i;
        int brow;
        const __bf16* base;
        if (EPI == EPI_SWIGLU) {
          base = (r < BN / 2) ? B0 : B1;
          brow = n0 + ((r < BN / 2) ? r : r - BN / 2);
        } else {
          base = B0;
          brow = n0 + r;
        }
        b_src[i] = (brow < p.N) ? base + (size_t)brow * K + cchunk * 8 : nullptr;
      }
    }

    // fragments with at least one valid row
    const int fm_active = max(0, min(FM, (rows - wm * WTM + 31) / 32));

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    i32x4 ra[A_CH], rb[B_CH];
    auto gload = [&](int ks) {
      const size_t koff = (size_t)ks * 64;
#pragma unroll
      for (int i = 0; i < A_CH; ++i)
        ra[i] = a_src[i] ? *reinterpret_cast<const i32x4*>(a_src[i] + koff) : i32x4{0, 0, 0, 0};
#pragma unroll
      for (int i = 0; i < B_CH; ++i)
        rb[i] = b_src[i] ? *reinterpret_cast<const i32x4*>(b_src[i] + koff) : i32x4{0, 0, 0, 0};
    };
    auto lstore = [&](int buf) {
      char* as = As + buf * BM * 128;
      char* bs = Bs + buf * BN * 128;
#pragma unroll
      for (int i = 0; i < A_CH; ++i)
        *reinterpret_cast<i32x4*>(as + lds_off(rbase + 32 * i, cchunk)) = ra[i];
#pragma unroll
      for (int i = 0; i < B_CH; ++i)
        *reinterpret_cast<i32x4*>(bs + lds_off(rbase + 32 * i, cchunk)) = rb[i];
    };

    // LDS row of B fragment j for this wave
    auto brow_of = [&](int j) -> int {
      if (EPI == EPI_SWIGLU)
        return (j < FN / 2) ? wn * (WTN / 2) + 32 * j : BN / 2 + wn * (WTN / 2) + 32 * (j - FN / 2);
      return wn * WTN + 32 * j;
    };

    gload(0);
    __syncthreads();  // previous tile's readers are done with the LDS
    lstore(0);
    __syncthreads();

    for (int ks = 0; ks < nk; ++ks) {
      const int buf = ks & 1;
      if (ks + 1 < nk) gload(ks + 1);
      const char* as = As + buf * BM * 128;
      const char* bs = Bs + buf * BN * 128;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int ch = 2 * kk + (lane >> 5);
        i32x4 bfr[FN];
#pragma unroll
        for (int j = 0; j < FN; ++j)
          bfr[j] = *reinterpret_cast<const i32x4*>(bs + lds_off(brow_of(j) + (lane & 31), ch));
#pragma unroll
        for (int i = 0; i < FM; ++i) {
          if (i < fm_active) {
            const i32x4 afr =
                *reinterpret_cast<const i32x4*>(as + lds_off(wm * WTM + 32 * i + (lane & 31), ch));
#pragma unroll
            for (int j = 0; j < FN; ++j)
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                  __builtin_bit_cast(bf16x8, afr), __builtin_bit_cast(bf16x8, bfr[j]), acc[i][j], 0, 0, 0);
          }
        }
      }
      if (ks + 1 < nk) lstore(buf ^ 1);
      __syncthreads();
    }

    // ---- epilogue ---------------------------------------------------------
    OutT* const C = static_cast<OutT*>(p.C);
    const size_t ldc = (size_t)p.ldc;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      if (i >= fm_active) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = wm * WTM + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (row >= rows) continue;
        const size_t crow = (size_t)(row0 + row) * ldc;
        if (EPI == EPI_SWIGLU) {
#pragma unroll
          for (int j = 0; j < FN / 2; ++j) {
            const int col = n0 + wn * (WTN / 2) + 32 * j + (lane & 31);
            if (col < p.N) store_out(C, crow + col, silu_f(acc[i][j][r]) * acc[i][j + FN / 2][r]);
          }
        } else {
#pragma unroll
          for (int j = 0; j < FN; ++j) {
            const int col = n0 + wn * WTN + 32 * j + (lane & 31);
            if (col < p.N) store_out(C, crow + col, acc[i][j][r]);
          }
        }
      }
    }
  }
}

struct LaunchInfo {
  int occupancy = 0;
};

template <int BM, int BN, int WGM, int WGN, int EPI, bool OUT_F32>
hipError_t launch_cfg(const GemmProblem& p, hipStream_t s) {
  auto kern = gemm_bf16_kernel<BM, BN, WGM, WGN, EPI, OUT_F32>;
  constexpr size_t lds = (size_t)2 * (BM + BN) * 128;
  static std::once_flag once;
  static int occ = 1;
  static hipError_t init_err = hipSuccess;
  std::call_once(once, [&] {
    init_err = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (init_err == hipSuccess) {
      int o = 0;
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&o, kern, kThreads, lds) == hipSuccess && o > 0) occ = o;
    }
  });
  if (init_err != hipSuccess) return init_err;
  const int ncols_tile = (EPI == EPI_SWIGLU) ? BN / 2 : BN;
  const long long nt = (p.N + ncols_tile - 1) / ncols_tile;
  const int groups = p.offsets ? p.groups : 1;
  // upper bound on m-tiles: every non-empty group adds at most one partial tile
  const long long mt_upper = (p.M + BM - 1) / BM + (p.offsets ? groups : 0);
  const long long upper = mt_upper * nt;
  if (upper <= 0) return hipSuccess;
  long long grid = (long long)device_cu_count() * occ;
  if (grid > upper) grid = upper;
  if (grid >= 8) grid -= grid % 8;
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kThreads), lds, s, p);
  return hipGetLastError();
}

template <int BM, int BN, int WGM, int WGN>
hipError_t launch_epi(const GemmProblem& p, int epi, bool out_f32, hipStream_t s) {
  if (epi == EPI_SWIGLU) return launch_cfg<BM, BN, WGM, WGN, EPI_SWIGLU, false>(p, s);
  if (out_f32) return launch_cfg<BM, BN, WGM, WGN, EPI_STORE, true>(p, s);
  return launch_cfg<BM, BN, WGM, WGN, EPI_STORE, false>(p, s);
}

}  // namespace

hipError_t launch_gemm_bf16(const GemmProblem& p, int epi, bool out_f32, hipStream_t s) {
  if (p.M <= 0 || p.N <= 0) return hipSuccess;
  const int groups = p.offsets ? p.groups : 1;
  const double avg_rows = (double)p.M / groups;
  if (avg_rows >= 512) return launch_epi<256, 256, 2, 2>(p, epi, out_f32, s);
  if (avg_rows >= 64) return launch_epi<128, 256, 2, 2>(p, epi, out_f32, s);
  if (avg_rows >= 24) return launch_epi<64, 128, 2, 2>(p, epi, out_f32, s);
  return launch_epi<32, 256, 1, 4>(p, epi, out_f32, s);
}

}  // namespace moe
