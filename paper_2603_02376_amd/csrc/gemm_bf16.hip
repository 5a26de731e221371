// Grouped bf16 GEMM on the gfx950 matrix cores (v_mfma_f32_32x32x16_bf16).
//
// This is the expert FFN of the MoE layer (App. M step 3; App. F GEMM1 +
// SwiGLU + GEMM2): every expert multiplies its segment of dispatched token
// rows by its own weight matrix. One kernel covers
//   * GEMM1 with the SwiGLU epilogue: h = silu(X·Wgᵀ) * (X·Wuᵀ), the gate and
//     up columns of one output column sitting in the same lane and register,
//   * GEMM2 and the router GEMM: C = X·Wᵀ (bf16 or fp32 output, optionally
//     split along K into fp32 partial sums),
// with the token gather (row r reads x[sorted_token[r]]) fused into the
// A-tile load, so the permuted activations are never materialised.
//
// Structure
//   * Persistent grid: each workgroup walks tiles tile = vb, vb+G, ...; the
//     tile list (k-split, expert, m-tile, n-tile) is derived in the prologue
//     from the expert offsets, so no host round trip is needed and empty
//     experts cost nothing. vb is the XCD-aware virtual block id: workgroups
//     are handed to the 8 XCDs round-robin, so vb = (b % 8) * (G/8) + b/8
//     gives every XCD a contiguous run of tiles, i.e. the tiles of one expert
//     share that XCD's L2 (A rows are re-read by every n-tile, B columns by
//     every m-tile).
//   * Within an expert, tiles are ordered in groups of kGroupM m-tiles per
//     n-tile so that m-tiles sharing a B slice run side by side.
//   * K is walked in steps of BK (64: 128 bytes per row) through a ring of
//     LDS slots filled by direct global->LDS loads (global_load_lds_dwordx4):
//     no register staging, and all but one slot of loads stay in flight while
//     the matrix cores work on the current slot. A step waits only for its own
//     loads (s_waitcnt vmcnt(n), counting the younger steps still in flight),
//     then one workgroup barrier makes every wave's loads visible and frees
//     the slot read in the previous step for refilling. The ring fills a
//     fixed LDS budget: a tile whose segment has at most 128 rows loads only
//     128 A rows per step and so gets more slots (3 instead of 2 at 256x256).
//   * LDS rows are 128 bytes; the 16-byte chunk c of row r lives at chunk
//     c ^ (r & 7). A direct load writes 64 lanes x 16 B contiguously, i.e. 8
//     rows, so lane l fetches the global chunk (l & 7) ^ (l >> 3) of its row:
//     the swizzle is applied on the global side, the loads stay fully
//     coalesced (one 128-byte row per 8 lanes), and the column-wise fragment
//     reads (8 rows, same chunk) are bank-conflict free.
//   * 4 or 8 waves per workgroup in a WGM x WGN grid; a wave owns FM x FN
//     32x32 accumulators; fragment i of wave row wm covers rows
//     (wm + WGM*i)*32.., so a segment shorter than the tile still keeps every
//     SIMD busy. With 8 waves two waves share each SIMD, so one
//     wave's LDS reads and barrier waits overlap the other's MFMAs; within a
//     wave the fragments of the next k sub-step are read while the MFMAs of
//     the current one run. Fragments whose 32 rows all lie past the segment's end are
//     skipped (wave-uniform), so short expert segments do not pay for the
//     padding. Rows past the end are loaded from the segment's last row (the
//     count of loads per step stays fixed, as the waits require) and never
//     stored.
#include "moe_internal.h"

#include <mutex>
#include <type_traits>

namespace moe {
namespace {

constexpr int kGroupM = 4;

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef __attribute__((address_space(1))) void* gbl_ptr_t;

// LDS byte offset of 16-byte chunk `chunk` of tile row `row`, for rows of
// ROWB = 2*BK bytes (128 or 64). The chunk index is XORed with a function of
// the row so that 8 consecutive rows read at the same logical chunk hit 8
// distinct 16-byte bank groups (rows of 64 bytes pair up within 128 bytes).
template <int ROWB>
__device__ __forceinline__ int lds_off(int row, int chunk) {
  if constexpr (ROWB == 128) return (row << 7) + ((chunk ^ (row & 7)) << 4);
  else return (row << 6) + ((chunk ^ ((row >> 1) & 3)) << 4);
}

__device__ __forceinline__ float silu_f(float g) { return g / (1.0f + __expf(-g)); }

__device__ __forceinline__ void store_out(__bf16* C, size_t i, float v) { C[i] = static_cast<__bf16>(v); }
__device__ __forceinline__ void store_out(float* C, size_t i, float v) { C[i] = v; }

// 16-byte direct load from global memory into LDS: lane l of the wave writes
// lds_base + 16*l.
__device__ __forceinline__ void dma16(const void* g, void* lds_base) {
  __builtin_amdgcn_global_load_lds((gbl_ptr_t)(g), (lds_ptr_t)(lds_base), 16, 0, 0);
}

// Wait until at most N vector-memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Workgroup barrier ordering LDS accesses only (no wait on global traffic).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Exclusive scan of one int per thread over a block of NW waves; returns the
// exclusive prefix and writes the block total to *total.
template <int NW>
__device__ int block_exclusive_scan(int v, int* scratch /*[NW]*/, int* total) {
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
  for (int w = 0; w < NW; ++w) {
    int s = scratch[w];
    if (w < wave) base += s;
    tot += s;
  }
  *total = tot;
  return base + inc - v;
}

// Calls f(std::integral_constant<int, n>) for a runtime n in [0, N].
template <int N, typename F>
__device__ __forceinline__ void with_count(int n, F&& f) {
  if constexpr (N == 0) {
    f(std::integral_constant<int, 0>{});
  } else {
    if (n == N) f(std::integral_constant<int, N>{});
    else with_count<N - 1>(n, f);
  }
}

// LDS budget of the stage ring (the kernel's static LDS takes ~1 KB more).
constexpr int kLdsRing = 144 * 1024;

template <int BM, int BN, int BK, int WGM, int WGN, int EPI, bool OUT_F32>
__global__ void __launch_bounds__(64 * WGM * WGN)
gemm_bf16_kernel(GemmProblem p) {
  constexpr int NW = WGM * WGN;                  // waves per workgroup
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int FM = WTM / 32, FN = WTN / 32;
  constexpr int ROWB = 2 * BK;                   // LDS bytes per tile row
  constexpr int CPR = BK / 8;                    // 16-byte chunks per row
  constexpr int RPI = 1024 / ROWB;               // rows written by one direct load of a wave
  constexpr int RPR = RPI * NW;                  // rows written by one round of direct loads
  constexpr int B_CH = BN / RPR;                 // direct B loads per wave per step
  static_assert(BK == 64 || BK == 32, "k step");
  static_assert(NW == 4 || NW == 8, "4 or 8 waves");
  static_assert(BM % RPR == 0 && BN % RPR == 0, "whole rounds of direct loads");
  static_assert(EPI != EPI_SWIGLU || (BN / 2) % RPR == 0, "gate and up rows in separate rounds");
  static_assert(FM >= 1 && FN >= 1 && WTM % 32 == 0 && WTN % 32 == 0, "32x32 fragments");
  static_assert(EPI != EPI_SWIGLU || (FN % 2 == 0 && B_CH % 2 == 0), "swiglu pairs gate/up fragments");
  using OutT = typename std::conditional<OUT_F32, float, __bf16>::type;

  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ int tstart[257];
  __shared__ int scan_scratch[NW];

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
    const int ex = block_exclusive_scan<NW>(mt, scan_scratch, &total);
    if (tid < groups) tstart[tid] = ex;
    if (tid == 0) tstart[groups] = total;
    __syncthreads();
  }
  const int ncols_tile = (EPI == EPI_SWIGLU) ? BN / 2 : BN;
  const int Nt = (p.N + ncols_tile - 1) / ncols_tile;
  const int tiles_per_split = tstart[groups] * Nt;
  const int ksplit = max(p.ksplit, 1);
  const int nk_all = p.K / BK;
  const int kq = (nk_all + ksplit - 1) / ksplit;  // k-steps per split
  const int total_tiles = tiles_per_split * ksplit;

  const int G = gridDim.x;
  const int b = blockIdx.x;
  const int vb = (G % 8 == 0) ? (b % 8) * (G / 8) + (b / 8) : b;

  const __bf16* const A = static_cast<const __bf16*>(p.A);
  const size_t K = (size_t)p.K;

  // this lane's place in a direct load: row lr of the RPI-row group, fetching
  // logical chunk lc so that it lands in physical chunk (lane % CPR)
  const int lr = lane / CPR;
  const int lc = (ROWB == 128) ? ((lane & 7) ^ lr) : ((lane & 3) ^ ((lr >> 1) & 3));

  // LDS row of B fragment j for this wave
  auto brow_of = [&](int j) -> int {
    if (EPI == EPI_SWIGLU)
      return (j < FN / 2) ? wn * (WTN / 2) + 32 * j : BN / 2 + wn * (WTN / 2) + 32 * (j - FN / 2);
    return wn * WTN + 32 * j;
  };

  for (int tile_all = vb; tile_all < total_tiles; tile_all += G) {
    // ---- decode the tile --------------------------------------------------
    const int split = tile_all / tiles_per_split;
    const int tile = tile_all - split * tiles_per_split;
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
    const int ks0 = split * kq;
    const int nk = max(0, min(nk_all, ks0 + kq) - ks0);

    // ---- per-lane B sources (element pointers at k = ks0*BK) ---------------
    const __bf16* b_src[B_CH];
    {
      const size_t gstride = (size_t)p.N * K;
      const __bf16* B0 = static_cast<const __bf16*>(p.B0) + (size_t)e * gstride;
      const __bf16* B1 = (EPI == EPI_SWIGLU) ? static_cast<const __bf16*>(p.B1) + (size_t)e * gstride : nullptr;
#pragma unroll
      for (int i = 0; i < B_CH; ++i) {
        const int r = i * RPR + wave * RPI + lr;
        const __bf16* base = B0;
        int brow = n0 + r;
        if (EPI == EPI_SWIGLU && i >= B_CH / 2) {  // second half of the tile: up rows
          base = B1;
          brow = n0 + r - BN / 2;
        }
        brow = min(brow, p.N - 1);
        b_src[i] = base + (size_t)brow * K + (size_t)ks0 * BK + lc * 8;
      }
    }

    // fragment i of wave row wm covers rows [(wm + WGM*i)*32, +32): the valid
    // rows of a short segment spread over every wave row (and SIMD)
    int fm_count = 0;
#pragma unroll
    for (int i = 0; i < FM; ++i) fm_count += ((wm + WGM * i) * 32 < rows) ? 1 : 0;
    const int fm_active = __builtin_amdgcn_readfirstlane(fm_count);

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // The K loop for an A tile of AR rows (AR = BM, or 128 when the segment's
    // rows fit: fewer direct loads per step and a deeper LDS ring).
    auto body = [&](auto ar_c) {
      constexpr int AR = decltype(ar_c)::value;
      constexpr int A_CH = AR / RPR;
      constexpr int LOADS = A_CH + B_CH;
      constexpr int SLOT = (AR + BN) * ROWB;
      constexpr int STAGES = (kLdsRing / SLOT) < 4 ? (kLdsRing / SLOT) : 4;
      static_assert(AR % RPR == 0 && STAGES >= 2 && LOADS * (STAGES - 2) < 64, "pipeline shape");

      const __bf16* a_src[A_CH];
#pragma unroll
      for (int i = 0; i < A_CH; ++i) {
        const int r = min(i * RPR + wave * RPI + lr, rows - 1);
        const int ar = p.gather ? min(max(p.gather[row0 + r], 0), p.a_rows - 1) : row0 + r;
        a_src[i] = A + (size_t)ar * K + (size_t)ks0 * BK + lc * 8;
      }
      auto issue = [&](int ks, int slot) {
        char* as = smem + slot * SLOT;
        char* bs = as + AR * ROWB;
        const size_t koff = (size_t)ks * BK;
#pragma unroll
        for (int i = 0; i < A_CH; ++i) dma16(a_src[i] + koff, as + (i * RPR + wave * RPI) * ROWB);
#pragma unroll
        for (int i = 0; i < B_CH; ++i) dma16(b_src[i] + koff, bs + (i * RPR + wave * RPI) * ROWB);
      };

      lds_barrier();  // every wave is done reading the previous tile's slots
#pragma unroll
      for (int s = 0; s < STAGES - 1; ++s)
        if (s < nk) issue(s, s);

      // compiled once per count of active A fragments so that the MFMA
      // stream has no branches (every wave runs the same barriers)
      auto kloop = [&](auto nact_c) {
        constexpr int NACT = decltype(nact_c)::value;
        for (int ks = 0; ks < nk; ++ks) {
          // wait for this step's loads; younger steps may stay in flight
          const int younger = min(STAGES - 2, nk - 1 - ks);
          if (STAGES >= 4 && younger >= 2) wait_vmcnt<(STAGES >= 4 ? 2 * LOADS : 0)>();
          else if (STAGES >= 3 && younger >= 1) wait_vmcnt<(STAGES >= 3 ? LOADS : 0)>();
          else wait_vmcnt<0>();
          lds_barrier();
          if (ks + STAGES - 1 < nk) issue(ks + STAGES - 1, (ks + STAGES - 1) % STAGES);
          if constexpr (NACT > 0) {
            const char* as = smem + (ks % STAGES) * SLOT;
            const char* bs = as + AR * ROWB;
            // fragments of sub-step kk+1 are read while the MFMAs of kk run
            i32x4 af[2][NACT], bf[2][FN];
            auto read_frags = [&](int kk, int sel) {
              const int ch = 2 * kk + (lane >> 5);
#pragma unroll
              for (int j = 0; j < FN; ++j)
                bf[sel][j] = *reinterpret_cast<const i32x4*>(bs + lds_off<ROWB>(brow_of(j) + (lane & 31), ch));
#pragma unroll
              for (int i = 0; i < NACT; ++i)
                af[sel][i] =
                    *reinterpret_cast<const i32x4*>(as + lds_off<ROWB>((wm + WGM * i) * 32 + (lane & 31), ch));
            };
            read_frags(0, 0);
#pragma unroll
            for (int kk = 0; kk < BK / 16; ++kk) {
              if (kk + 1 < BK / 16) read_frags(kk + 1, (kk + 1) & 1);
#pragma unroll
              for (int i = 0; i < NACT; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                  acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, af[kk & 1][i]),
                                                                      __builtin_bit_cast(bf16x8, bf[kk & 1][j]),
                                                                      acc[i][j], 0, 0, 0);
            }
          }
        }
      };
      // fragments of rows >= AR are never active
      constexpr int FMA = (AR / 32 + WGM - 1) / WGM < FM ? (AR / 32 + WGM - 1) / WGM : FM;
      with_count<FMA>(min(fm_active, FMA), kloop);
    };
    if constexpr (BM > 128) {
      if (rows <= 128) body(std::integral_constant<int, 128>{});
      else body(std::integral_constant<int, BM>{});
    } else {
      body(std::integral_constant<int, BM>{});
    }

    // ---- epilogue ---------------------------------------------------------
    OutT* const C = static_cast<OutT*>(p.C) + (size_t)split * p.c_split_stride;
    const size_t ldc = (size_t)p.ldc;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      if (i >= fm_active) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = (wm + WGM * i) * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
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

template <int BM, int BN, int BK, int WGM, int WGN, int EPI, bool OUT_F32>
hipError_t launch_cfg(const GemmProblem& p, hipStream_t s) {
  auto kern = gemm_bf16_kernel<BM, BN, BK, WGM, WGN, EPI, OUT_F32>;
  constexpr size_t lds = kLdsRing;
  const hipError_t init_err = set_dynamic_lds((const void*)kern, (int)lds);
  if (init_err != hipSuccess) return init_err;
  static std::once_flag once;  // the occupancy is the same on every gfx950 device
  static int occ = 1;
  std::call_once(once, [&] {
    int o = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&o, kern, 64 * WGM * WGN, lds) == hipSuccess && o > 0) occ = o;
  });
  const int ncols_tile = (EPI == EPI_SWIGLU) ? BN / 2 : BN;
  const long long nt = (p.N + ncols_tile - 1) / ncols_tile;
  const int groups = p.offsets ? p.groups : 1;
  // upper bound on m-tiles: every non-empty group adds at most one partial tile
  const long long mt_upper = (p.M + BM - 1) / BM + (p.offsets ? groups : 0);
  const long long upper = mt_upper * nt * (long long)(p.ksplit > 1 ? p.ksplit : 1);
  if (upper <= 0) return hipSuccess;
  long long grid = (long long)device_cu_count() * occ;
  if (grid > upper) grid = upper;
  if (grid >= 8) grid -= grid % 8;
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(64 * WGM * WGN), lds, s, p);
  return hipGetLastError();
}

template <int BM, int BN, int BK, int WGM, int WGN>
hipError_t launch_epi(const GemmProblem& p, int epi, bool out_f32, hipStream_t s) {
  if (epi == EPI_SWIGLU) return launch_cfg<BM, BN, BK, WGM, WGN, EPI_SWIGLU, false>(p, s);
  if (out_f32) return launch_cfg<BM, BN, BK, WGM, WGN, EPI_STORE, true>(p, s);
  return launch_cfg<BM, BN, BK, WGM, WGN, EPI_STORE, false>(p, s);
}

}  // namespace

hipError_t launch_gemm_bf16(const GemmProblem& p, int epi, bool out_f32, hipStream_t s) {
  if (p.M <= 0 || p.N <= 0) return hipSuccess;
  if (p.tile == GEMM_TILE_SKINNY) return launch_epi<32, 256, 64, 1, 4>(p, epi, out_f32, s);
  if (p.tile == GEMM_TILE_M64) return launch_epi<64, 256, 64, 1, 4>(p, epi, out_f32, s);
  const int groups = p.offsets ? p.groups : 1;
  const double avg_rows = (double)p.M / groups;
  if (avg_rows >= 64) return launch_epi<256, 256, 64, 4, 2>(p, epi, out_f32, s);
  if (avg_rows >= 24) return launch_epi<64, 256, 64, 1, 4>(p, epi, out_f32, s);
  return launch_epi<32, 256, 64, 1, 4>(p, epi, out_f32, s);
}

}  // namespace moe
