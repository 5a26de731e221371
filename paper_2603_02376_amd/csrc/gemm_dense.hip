// Compute-bound grouped bf16 GEMM over packed expert weights (gfx950).
//
// The expert FFN of the MoE layer (App. M step 3; App. F GEMM1 + SwiGLU +
// GEMM2) when every expert holds many token rows: at the Mixtral shape
// (~1,024 rows per expert) each weight byte feeds ~1,000 FLOP, far above the
// MI355X ridge, so the kernel is organised around the matrix cores rather
// than around the weight stream (gemm_stream.hip, for the weight-bound
// DeepSeek-V3 shape):
//
//   * Output tiles of 256 token rows x 256 weight columns (GEMM1: 128 h
//     columns with their gate and up rows; GEMM2: 256 output columns), one
//     workgroup of 8 waves per compute unit (two per SIMD, so one wave's LDS
//     and barrier waits are covered by the other's MFMAs), each wave 128
//     token rows x 64 weight columns (32 accumulator tiles of 16x16). A K
//     step of 32 feeds every wave 32 MFMAs (v_mfma_f32_16x16x32_bf16) from
//     12 fragment reads: the same operand bytes and matrix-core cycles as
//     the 32x32x16 form, but the chip holds a higher clock under it (it
//     runs at its power limit here, and this instruction costs less energy
//     per FLOP).
//   * Both operands go through a 4-slot LDS ring of 32 KB (16 KB of token
//     rows, 16 KB of weights per step) filled by direct global->LDS loads
//     (buffer_load_dwordx4 ... lds): no register staging, loads issued three
//     steps ahead and spread between the MFMAs. The weights are one
//     contiguous 16 KB run per step in the packed layout (moe_pack_weights),
//     already in the lane order of the MFMA operand; the token rows are
//     gathered through sorted_token, 16-byte chunks XOR-swizzled on the global
//     side so the fragment reads are bank-conflict free.
//   * At the end of step x every wave waits for its own loads of step x+2 and
//     meets the others at one barrier, which publishes step x+2 and frees the
//     slot read in step x; the first token fragment and the weight fragments
//     of step x+1 (published a step earlier) are read before that barrier, so
//     no LDS latency sits between a barrier and the MFMAs. Only direct loads write the ring during the K
//     loop, so the hand-written vmcnt waits are exact.
//   * Rows: an expert's segment is cut into full 256-row blocks plus one
//     remainder block; 32-row fragments alternate between the two wave rows,
//     so a short block keeps both busy. The K loop is compiled per count of
//     active fragments (no branches in the MFMA stream).
//   * Schedule: a persistent grid, one workgroup per compute unit, tiles
//     dealt XCD-aware: each XCD takes runs of 32 consecutive tiles, which
//     are 8 column tiles x the m-blocks of one expert, so the m-blocks of a
//     column tile share its weights and the column tiles share the token rows
//     through that XCD's L2.
//   * Epilogue: the SwiGLU (GEMM1) in registers, the tile assembled in LDS and
//     written in whole 128-byte lines.
#include "moe_internal.h"

#include <algorithm>
#include <type_traits>
#include <utility>

namespace moe {
namespace {

typedef __attribute__((address_space(3))) void* lds_ptr_t;

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kBM = 256;                       // token rows per tile
constexpr int kBK = 32;                        // K per pipeline step
constexpr int kSlots = 4;                      // LDS ring slots
constexpr int kABytes = kBM * kBK * 2;         // 16 KB of token rows per step
constexpr int kSlotBytes = 2 * kABytes;        // + 16 KB of weights
constexpr int kRing = kSlots * kSlotBytes;     // 128 KB
constexpr int kNtGroup = 8;                    // column tiles per run of one expert
constexpr int kStreamStore = 19;               // output stores: sc0 sc1 nt

// Minimum average rows per group for this kernel (below it the weight stream
// is the bound and gemm_stream is used).
constexpr int kDenseMinAvgRows = 512;

// K split of the short remainder blocks of GEMM2. A remainder block of at
// most 192 rows streams a column tile's whole K range of weights for a few
// rows; with a long K (Mixtral: 14336, two rounds of full 256-row tiles of
// ~365 us each) the remainder tiles make a third round on a quarter of the
// compute units. Each such tile is cut into kPartKs tiles over consecutive
// quarters of K that write fp32 partial sums (up to kPartRows rows x 256
// columns each) to a workspace; dense_part_reduce_kernel then adds the
// quarters in order (a fixed order: the result does not depend on which
// workgroup ran which quarter when) and writes the bf16 rows.
constexpr int kPartKs = 4;
constexpr int kPartRows = 192;                 // rows of a section-2 (remainder) block, at most
constexpr int kPartMetaBytes = 4096;           // [0]: remainder blocks, [1 + i]: group of block i
constexpr size_t kPartBudget = (size_t)256 << 20;

template <typename F, int... Is>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, Is...>) {
  (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// f(std::integral_constant<int, n>) for a runtime n in [0, N].
template <int N, typename F>
__device__ __forceinline__ void with_count(int n, F&& f) {
  if constexpr (N == 0) {
    f(std::integral_constant<int, 0>{});
  } else {
    if (n == N) f(std::integral_constant<int, N>{});
    else with_count<N - 1>(n, f);
  }
}

// Token-row region of a slot: 64-byte rows, 16-byte chunk c of row r at
// chunk c ^ ((r >> 2) & 3). The LDS serves a 16-byte read 16 lanes at a
// time from a 256-byte window of banks; the 16 consecutive rows those lanes
// read at one logical chunk then fall on 16 distinct 16-byte bank groups
// (4 (r % 4) + physical chunk).
__device__ __forceinline__ int a_off(int row, int chunk) { return (row << 6) + ((chunk ^ ((row >> 2) & 3)) << 4); }
__device__ __forceinline__ float silu_f(float g) { return g / (1.0f + __expf(-g)); }

__device__ __forceinline__ int block_scan(int v, int* scratch, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int n = __shfl_up(inc, o, 64);
    if (lane >= o) inc += n;
  }
  __syncthreads();  // the previous scan's reads of scratch are done
  if (lane == 63) scratch[wave] = inc;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const int s = scratch[w];
    if (w < wave) base += s;
    tot += s;
  }
  *total = tot;
  return base + inc - v;
}

// EPI_SWIGLU: GEMM1 (weight columns = 128 h columns x gate/up);
// EPI_STORE:  GEMM2 (256 output columns).
template <int EPI>
__global__ void __launch_bounds__(kThreads, 1) gemm_dense_kernel(GemmProblem p) {
  constexpr int TCOLS = (EPI == EPI_SWIGLU) ? 128 : 256;  // output columns per tile
  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ int tstart[257];  // section 1: first m-block of each group
  __shared__ int rgroup[256];  // section 2: group of each remainder block, in order
  __shared__ int n_rgroup;
  __shared__ int scan_scratch[kWaves];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: LDS load targets stay scalar
  const int wm = wave >> 2, wn = wave & 3;  // wave row (token rows), wave column (packed weight slot)
  const int groups = p.offsets ? p.groups : 1;
  // Tile order. A group of c rows has c / 256 full blocks and a remainder of
  // c % 256 rows whose cost (MFMAs of its busier wave row) is a fraction of a
  // full block's. Section 1 holds every block that costs as much as a full
  // one (full blocks and remainders of more than 192 rows), group by group;
  // section 2 the cheaper remainders, costliest first. With the persistent
  // grid dealing tiles round-robin, the cheap tiles fill the last round
  // instead of adding a round of their own.
  auto group_rows = [&](int g) {
    if (!p.offsets) return p.M;
    const int lo = min(max(p.offsets[g], 0), p.M);
    return min(max(p.offsets[g + 1], lo), p.M) - lo;
  };
  auto rem_class = [](int c) { return ((c % kBM + 31) / 32 + 1) / 2; };  // 0: none; 4: as costly as a full block
  {
    int mb = 0, cls = 0;
    if (tid < groups) {
      const int c = group_rows(tid);
      cls = rem_class(c);
      mb = c / kBM + (cls == 4 ? 1 : 0);
    }
    int total;
    const int ex = block_scan(mb, scan_scratch, &total);
    if (tid < groups) tstart[tid] = ex;
    if (tid == 0) tstart[groups] = total;
    // section 2 positions: classes 3, 2, 1 in turn, groups ascending within a class
    int base = 0;
    for (int c3 = 3; c3 >= 1; --c3) {
      int n;
      const int pos = block_scan(tid < groups && cls == c3 ? 1 : 0, scan_scratch, &n);
      if (tid < groups && cls == c3) rgroup[base + pos] = tid;
      base += n;
    }
    if (tid == 0) n_rgroup = base;
    __syncthreads();
  }
  const int Nt = p.N / TCOLS;
  const int tiles1 = tstart[groups] * Nt;
  // K parts of a section-2 tile (GEMM2 with a split workspace; nk % (4 KS) == 0, checked at launch)
  const int KS = (EPI == EPI_STORE && p.part_ks > 1) ? p.part_ks : 1;
  const int total_tiles = tiles1 + n_rgroup * Nt * KS;
  const int K = p.K, nk = K / kBK;  // nk % 4 == 0 (checked at launch)
  if (KS > 1 && blockIdx.x == 0) {  // the remainder blocks, for dense_part_reduce_kernel
    int32_t* const meta = static_cast<int32_t*>(p.dense_part);
    if (tid == 0) meta[0] = n_rgroup;
    if (tid < n_rgroup) meta[1 + tid] = rgroup[tid];
  }
  const int G = gridDim.x, b = blockIdx.x;
  const int vb = (G % 8 == 0) ? (b % 8) * (G / 8) + (b / 8) : b;

  // this lane's part of a token-row direct load: row (lane >> 2) of a 16-row
  // group, fetching logical chunk lc so that it lands at physical chunk lane & 3
  const int lc = (lane & 3) ^ ((lane >> 4) & 3);

  for (int tile = vb; tile < total_tiles; tile += G) {
    // ---- decode: group e, m-block mb, column tile nt (split: remainder block
    // ridx's K part `part`)
    int e, mb, nt, part = 0, ridx = 0;
    if (tile < tiles1) {
      const int q = tile / Nt;
      int lo = 0, hi = groups - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (tstart[mid] <= q) lo = mid; else hi = mid - 1;
      }
      e = lo;
      // runs of kNtGroup column tiles x the group's section-1 blocks
      const int MB = tstart[e + 1] - tstart[e];
      const int local = tile - tstart[e] * Nt;
      const int ntg = local / (MB * kNtGroup);
      const int rem = local - ntg * MB * kNtGroup;
      const int gsz = min(kNtGroup, Nt - ntg * kNtGroup);
      mb = rem / gsz;
      nt = ntg * kNtGroup + rem % gsz;
    } else {
      const int t2 = tile - tiles1;
      part = t2 % KS;  // the K parts of one (block, column tile) are adjacent
      ridx = t2 / KS;
      e = rgroup[ridx / Nt];
      nt = ridx % Nt;
      mb = group_rows(e) / kBM;
    }
    const int gbeg = p.offsets ? min(max(p.offsets[e], 0), p.M) : 0;
    const int gend = p.offsets ? min(max(p.offsets[e + 1], gbeg), p.M) : p.M;
    const int row0 = gbeg + mb * kBM;
    const int rows = min(kBM, gend - row0);
    const bool split = KS > 1 && tile >= tiles1;
    const int nkl = split ? nk / KS : nk;  // K steps of this tile, from step kx0
    const int kx0 = part * nkl;

    // token rows of this wave's direct loads (rows past the block re-read
    // its last row: a fixed count of loads per step, never stored)
    const __amdgpu_buffer_rsrc_t a_rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<void*>(p.A), (short)0, (int)(uint32_t)((size_t)p.a_rows * K * 2), 0x00020000);
    uint32_t a_voff[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r = min(i * 128 + wave * 16 + (lane >> 2), rows - 1);
      const int ar = p.gather ? min(max(p.gather[row0 + r], 0), p.a_rows - 1) : row0 + r;
      a_voff[i] = (uint32_t)ar * (uint32_t)(K * 2) + lc * 16;
    }
    // weights: the tile's packed stream, K/64 blocks of 32 KB; this wave
    // loads the four 1 KB pieces of packed wave slot w = wave of each step
    // (pieces (w, kk, j) of a 64-wide block at ((w * 4 + kk) * 2 + j) KB)
    const char* const b_tile =
        static_cast<const char*>(p.B0) + ((size_t)e * Nt + nt) * (size_t)(K / 64) * 32768;
    const __amdgpu_buffer_rsrc_t b_rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char*>(b_tile), (short)0, (int)(uint32_t)((size_t)(K / 64) * 32768), 0x00020000);
    const uint32_t b_voff = (uint32_t)(lane * 16 + ((wave >> 1) * 8 + 2 * (wave & 1)) * 1024);

    // Direct loads of step x into slot s: token rows i * 128 + wave * 16 +
    // lane / 4 (i < AL), and the wave's two 1 KB weight pieces 2 wave + n of
    // the 64-wide block x / 2, K slices 2 (x % 2) and 2 (x % 2) + 1.
    auto load_a = [&](int x, int s, int i) __attribute__((always_inline)) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(a_rs, (lds_ptr_t)(smem + s * kSlotBytes + (i * 128 + wave * 16) * 64), 16,
                                               (int)a_voff[i], (kx0 + x) * 64, 0, 0);
    };
    auto load_b = [&](int x, int s, int n) __attribute__((always_inline)) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          b_rs, (lds_ptr_t)(smem + s * kSlotBytes + kABytes + (wave * 2 + n) * 1024), 16, (int)(b_voff + n * 1024),
          ((kx0 + x) >> 1) * 32768 + ((kx0 + x) & 1) * 4096, 0, 0);
    };

    // acc[f][wc]: 16 token rows (fragment f) x 16 weight columns (fragment wc)
    f32x4 acc[8][4];
#pragma unroll
    for (int f = 0; f < 8; ++f)
#pragma unroll
      for (int wc = 0; wc < 4; ++wc)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[f][wc][r] = 0.f;
    // active 32-row fragments of this wave: fragment i covers rows (wm + 2 i) * 32 ..
    const int nfrag = (rows + 31) / 32;
    const int nact = __builtin_amdgcn_readfirstlane((nfrag - wm + 1) / 2);

    // AL: token-row loads per wave and step (1 when the block has at most
    // 128 rows: the second half of the A region is never read)
    auto kloop = [&](auto nact_c, auto al_c) __attribute__((always_inline)) {
      constexpr int NACT = decltype(nact_c)::value, AL = decltype(al_c)::value;
      constexpr int LOADS = AL + 2;
      asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");  // the previous tile's LDS reads are done
      auto load_step = [&](int x, int s) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < AL; ++i) load_a(x, s, i);
#pragma unroll
        for (int n = 0; n < 2; ++n) load_b(x, s, n);
      };
      load_step(0, 0);
      load_step(1, 1);
      load_step(2, 2);
      // Fragments of v_mfma_f32_16x16x32_bf16 (weights as the first operand:
      // lane l supplies weight column l % 16, token row l % 16, and the 8 K
      // values 8 (l / 16) .. + 7 of the 32-wide step). Token fragment f: rows
      // (wm + 2 (f / 2)) * 32 + (f % 2) * 16 + 0..15; weight fragment wc:
      // columns (wc % 2) * 16 + 0..15 of j = wc / 2 (gate / up, or column
      // half) of packed wave slot wn.
      constexpr int NF = 2 * NACT;
      i32x4 wf[4], tf[2];  // weight fragments; a ring of token fragments
      auto read_t = [&](int s, int f) __attribute__((always_inline)) {
        return *reinterpret_cast<const i32x4*>(smem + s * kSlotBytes +
                                               a_off((wm + 2 * (f >> 1)) * 32 + (f & 1) * 16 + (lane & 15), lane >> 4));
      };
      // the packed 1 KB block (wn, K slice k, j) holds column c, K 8 h .. 8 h + 7 of the slice in lane 32 h + c
      auto read_w = [&](int s, int wc) __attribute__((always_inline)) {
        const int g = lane >> 4;  // K group: slice g / 2, half g % 2
        return *reinterpret_cast<const i32x4*>(smem + s * kSlotBytes + kABytes +
                                               (((wn * 2 + (g >> 1)) * 2 + (wc >> 1)) << 10) +
                                               ((g & 1) * 32 + (wc & 1) * 16 + (lane & 15)) * 16);
      };
      // Step x (slot U = x % 4): token fragment by token fragment, its four
      // MFMAs (one per weight fragment), the read of the next token fragment
      // (past the last one: the next step's first, PRE) and (LOAD)
      // a share of the loads of step x + 3 into slot (U + 3) % 4; with the
      // last token fragment each weight fragment, once its last MFMA is
      // issued, is replaced by the next step's (PRE). Token fragment f sits
      // in ring entry f % 2 (NF is even).
      // WAIT: 2 = wait for step x + 2's loads (younger: step x + 3's) then
      // barrier; 1 = wait for all loads then barrier; 0 = neither.
      auto step = [&](int x, auto u_c, auto load_c, auto pre_c, auto wait_c) __attribute__((always_inline)) {
        constexpr int U = decltype(u_c)::value;
        constexpr bool LOAD = decltype(load_c)::value, PRE = decltype(pre_c)::value;
        constexpr int WAIT = decltype(wait_c)::value;
        constexpr int LS = (U + 3) % kSlots;
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (NACT > 0) {
#pragma unroll
          for (int f = 0; f < NF; ++f) {
#pragma unroll
            for (int wc = 0; wc < 4; ++wc) {
              acc[f][wc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wf[wc]),
                                                                   __builtin_bit_cast(bf16x8, tf[f & 1]),
                                                                   acc[f][wc], 0, 0, 0);
              if (f == NF - 1 && PRE) wf[wc] = read_w((U + 1) % kSlots, wc);
            }
            if (f + 1 < NF) tf[(f + 1) & 1] = read_t(U, f + 1);
            else if (PRE) tf[0] = read_t((U + 1) % kSlots, 0);
            if constexpr (LOAD) {  // the step's loads, spread over the fragments
#pragma unroll
              for (int n = f * LOADS / NF; n < (f + 1) * LOADS / NF; ++n) {
                if (n < AL) load_a(x + 3, LS, n);
                else load_b(x + 3, LS, n - AL);
              }
            }
            __builtin_amdgcn_sched_barrier(0);
          }
        } else if constexpr (LOAD) {
          load_step(x + 3, LS);
        }
        if constexpr (WAIT == 2) asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(LOADS) : "memory");
        if constexpr (WAIT == 1) asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
        __builtin_amdgcn_sched_barrier(0);
      };
      using T_ = std::true_type;
      using F_ = std::false_type;
      using W2 = std::integral_constant<int, 2>;
      using W1 = std::integral_constant<int, 1>;
      using W0 = std::integral_constant<int, 0>;
      // steps 0 and 1 landed (step 2's loads may still fly); publish them
      asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(LOADS) : "memory");
      if constexpr (NACT > 0) {
#pragma unroll
        for (int wc = 0; wc < 4; ++wc) wf[wc] = read_w(0, wc);
        tf[0] = read_t(0, 0);
      }
      int x = 0;
      for (; x + 4 < nkl; x += 4)
        static_for<4>([&](auto u_c) { step(x + u_c, u_c, T_{}, T_{}, W2{}); });
      step(x, std::integral_constant<int, 0>{}, T_{}, T_{}, W2{});
      step(x + 1, std::integral_constant<int, 1>{}, F_{}, T_{}, W1{});
      step(x + 2, std::integral_constant<int, 2>{}, F_{}, T_{}, W0{});
      step(x + 3, std::integral_constant<int, 3>{}, F_{}, F_{}, W0{});
    };
    if (rows > 128) {
      with_count<4>(min(nact, 4), [&](auto n_c) { kloop(n_c, std::integral_constant<int, 2>{}); });
    } else {
      with_count<2>(min(nact, 2), [&](auto n_c) { kloop(n_c, std::integral_constant<int, 1>{}); });
    }

    if (split) {
      // fp32 partial sums of K part `part`: row r, output column c at
      // [(ridx KS + part) kPartRows + r] 256 + c (same register layout as below)
      float* const dst = reinterpret_cast<float*>(static_cast<char*>(p.dense_part) + kPartMetaBytes) +
                         ((size_t)ridx * KS + part) * (kPartRows * 256);
#pragma unroll
      for (int f = 0; f < 8; ++f) {
        if ((f >> 1) < nact) {
          const int r = (wm + 2 * (f >> 1)) * 32 + (f & 1) * 16 + (lane & 15);  // < kPartRows: at most 6 blocks
#pragma unroll
          for (int wc = 0; wc < 4; ++wc)  // columns (wc / 2) * 32 + (wc % 2) * 16 + 4 (lane / 16) + 0..3 of slot wn
            *reinterpret_cast<f32x4*>(dst + (size_t)r * 256 + wn * 64 + (wc >> 1) * 32 + (wc & 1) * 16 + 4 * (lane >> 4)) =
                acc[f][wc];
        }
      }
      continue;
    }
    // ---- epilogue. acc[f][wc] is the transposed 16x16 tile (weights were
    // the first MFMA operand): lane l holds token row l % 16 of fragment f and
    // weight columns 4 (l / 16) + 0..3 of fragment wc. Those 8-byte runs go
    // into an LDS copy of the output tile (rows of TCOLS bf16, 16-byte chunks
    // XOR-swizzled by row), which then leaves in whole rows, one 16-byte
    // chunk per thread, as streaming stores.
    {
      constexpr int OCH = TCOLS * 2 / 16;   // 16-byte chunks per output row
      constexpr int OROWS = kThreads / OCH; // rows per store pass
      asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");  // every wave is done with the ring
      const int hb = 8 * ((lane >> 4) & 1);  // byte offset of the 4-column run in its 16-byte chunk
#pragma unroll
      for (int f = 0; f < 8; ++f) {
        __builtin_amdgcn_sched_barrier(0);
        if ((f >> 1) < nact) {
          const int r = (wm + 2 * (f >> 1)) * 32 + (f & 1) * 16 + (lane & 15);
          char* const orow = smem + r * (TCOLS * 2);
          if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
            for (int q = 0; q < 2; ++q) {  // gate fragment q, up fragment 2 + q: h columns wn * 32 + q * 16 + 4 (l / 16)
              bf16x4 v;
#pragma unroll
              for (int c = 0; c < 4; ++c) v[c] = static_cast<__bf16>(silu_f(acc[f][q][c]) * acc[f][2 + q][c]);
              const int ch = wn * 4 + q * 2 + (lane >> 5);
              *reinterpret_cast<bf16x4*>(orow + ((ch ^ (r & (OCH - 1))) << 4) + hb) = v;
            }
          } else {
#pragma unroll
            for (int wc = 0; wc < 4; ++wc) {  // output columns wn * 64 + (wc / 2) * 32 + (wc % 2) * 16 + 4 (l / 16)
              bf16x4 v;
#pragma unroll
              for (int c = 0; c < 4; ++c) v[c] = static_cast<__bf16>(acc[f][wc][c]);
              const int ch = wn * 8 + (wc >> 1) * 4 + (wc & 1) * 2 + (lane >> 5);
              *reinterpret_cast<bf16x4*>(orow + ((ch ^ (r & (OCH - 1))) << 4) + hb) = v;
            }
          }
        }
      }
      asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
      const size_t ldc = (size_t)p.ldc;
      char* const cb = reinterpret_cast<char*>(p.C) + ((size_t)row0 * ldc + (size_t)nt * TCOLS) * 2;
      // rows >= `rows` fall outside the buffer range: the hardware drops them
      const __amdgpu_buffer_rsrc_t c_rs =
          __builtin_amdgcn_make_buffer_rsrc(cb, (short)0, (int)((uint32_t)rows * (uint32_t)(ldc * 2)), 0x00020000);
      const int oc = tid % OCH;
#pragma unroll
      for (int qp = 0; qp < kBM / OROWS; ++qp) {
        if (qp % 4 == 0) __builtin_amdgcn_sched_barrier(0);
        const int r = qp * OROWS + tid / OCH;
        if (r < rows) {
          const i32x4 v = *reinterpret_cast<const i32x4*>(smem + r * (TCOLS * 2) + ((oc ^ (r & (OCH - 1))) << 4));
          __builtin_amdgcn_raw_buffer_store_b128(v, c_rs, (int)((uint32_t)r * (uint32_t)(ldc * 2) + oc * 16), 0,
                                                 kStreamStore);
        }
      }
    }
  }
}

// Adds the kPartKs fp32 partial sums of every split remainder block in K
// order and writes its bf16 rows: one workgroup per (remainder block, column
// tile), one output column per thread.
__global__ void __launch_bounds__(256) dense_part_reduce_kernel(GemmProblem p) {
  const int Nt = p.N / 256;
  const int32_t* const meta = static_cast<const int32_t*>(p.dense_part);
  const int i = blockIdx.x / Nt, nt = blockIdx.x % Nt;
  if (i >= meta[0]) return;
  const int e = min(max(meta[1 + i], 0), p.groups - 1);
  const int gbeg = min(max(p.offsets[e], 0), p.M);
  const int gend = min(max(p.offsets[e + 1], gbeg), p.M);
  const int full = (gend - gbeg) / kBM * kBM;
  const int row0 = gbeg + full, rows = min(gend - gbeg - full, kPartRows);
  const float* const src = reinterpret_cast<const float*>(static_cast<const char*>(p.dense_part) + kPartMetaBytes) +
                           (size_t)(i * Nt + nt) * kPartKs * (kPartRows * 256);
  __bf16* const dst = static_cast<__bf16*>(p.C) + (size_t)nt * 256 + threadIdx.x;
  for (int r = 0; r < rows; ++r) {
    float acc = 0.f;
#pragma unroll
    for (int q = 0; q < kPartKs; ++q) acc += src[((size_t)q * kPartRows + r) * 256 + threadIdx.x];
    dst[(size_t)(row0 + r) * p.ldc] = static_cast<__bf16>(acc);
  }
}

size_t part_need(int groups, int nt) {
  return (size_t)kPartMetaBytes + (size_t)groups * nt * kPartKs * kPartRows * 256 * 4;
}

template <int EPI>
hipError_t launch_dense(const GemmProblem& p, hipStream_t s) {
  auto kern = gemm_dense_kernel<EPI>;
  const hipError_t init_err = set_dynamic_lds((const void*)kern, kRing);
  if (init_err != hipSuccess) return init_err;
  const int tcols = (EPI == EPI_SWIGLU) ? 128 : 256;
  const int groups = p.offsets ? p.groups : 1;
  GemmProblem q = p;
  q.part_ks = 1;
  if (EPI == EPI_STORE && p.offsets && p.dense_part) {
    const int nk = p.K / kBK;
    if (nk % (4 * kPartKs) == 0 && nk >= 256 && (size_t)p.dense_part_bytes >= part_need(groups, p.N / 256))
      q.part_ks = kPartKs;
  }
  const long long blocks_upper = (p.M + kBM - 1) / kBM + (p.offsets ? (long long)groups * q.part_ks : 0);
  const long long upper = blocks_upper * (p.N / tcols);
  if (upper <= 0) return hipSuccess;
  long long grid = device_cu_count();
  if (p.max_wg > 0 && grid > p.max_wg) grid = p.max_wg;
  if (grid > upper) grid = upper;
  if (grid >= 8) grid -= grid % 8;
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kThreads), kRing, s, q);
  if (q.part_ks > 1)
    hipLaunchKernelGGL(dense_part_reduce_kernel, dim3((unsigned)(groups * (p.N / 256))), dim3(256), 0, s, q);
  return hipGetLastError();
}

}  // namespace

size_t dense_part_bytes(int64_t rows, int32_t groups, int32_t n, int32_t k) {
  if (groups < 1 || groups > 256 || rows < (int64_t)kDenseMinAvgRows * groups) return 0;
  if (n <= 0 || n % 256 != 0 || k % 128 != 0 || (k / kBK) % (4 * kPartKs) != 0 || k / kBK < 256) return 0;
  const size_t need = part_need(groups, n / 256);
  return need <= kPartBudget ? need : 0;
}

bool gemm_dense_eligible(const GemmProblem& p) {
  if (p.a_scale || p.x_rows != 0 || p.seg_end || (p.offsets && !p.rows_exact)) return false;
  if (p.K % 128 != 0 || p.K < 256) return false;
  if ((size_t)p.a_rows * (size_t)p.K * 2 > 0xFFFFFFFFull || (size_t)(p.K / 64) * 32768 > 0x7FFFFFFFull) return false;
  const int groups = p.offsets ? p.groups : 1;
  return groups > 0 && groups <= 256 && (long long)p.M >= (long long)kDenseMinAvgRows * groups;
}

hipError_t launch_gemm_dense(const GemmProblem& p, int epi, hipStream_t s) {
  if (p.M <= 0 || p.N <= 0) return hipSuccess;
  if (!gemm_dense_eligible(p)) return hipErrorInvalidValue;
  if (epi == EPI_SWIGLU) return launch_dense<EPI_SWIGLU>(p, s);
  return launch_dense<EPI_STORE>(p, s);
}

}  // namespace moe
