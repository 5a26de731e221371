// Weight-streaming grouped bf16 GEMM over packed expert weights (gfx950).
// (GEMM1 also takes its token rows as per-token-scaled int8 or FP8 codes,
// converted to bf16 exactly while staged into LDS.)
//
// The expert FFN of the MoE layer (App. M step 3; App. F GEMM1 + SwiGLU +
// GEMM2) at DeepSeek-V3 shape is bound by reading every expert's weights
// once: ~128 tokens per expert give ~128 FLOP per weight byte, below the
// MI355X ridge. This kernel is organised around that stream:
//
//   * The weights are pre-packed (moe_pack_weights, once per model) so that a
//     workgroup's weights for one 64-wide K step are one contiguous 32 KB
//     block, already in the lane order of the MFMA B operand: each of the 4
//     waves reads its 8 KB as eight fully coalesced 1 KB loads straight into
//     registers. No LDS and no cross-wave sharing for B: waves own disjoint
//     output columns.
//   * Weights for kDepth-1 steps ahead stay in flight per wave (a ring of
//     register sets, the K loop unrolled so every set is statically indexed).
//     Two pipeline shapes: default (two steps in flight, passes of up to 192
//     rows) and deep (three steps in flight, passes of up to 160 rows, for
//     GEMM2 over small groups).
//   * The token rows (A, gathered through sorted_token) are shared by the 4
//     waves through an LDS ring of three or four slots: each wave loads its share of a
//     step's rows into registers three steps ahead and writes them to the
//     ring two steps ahead; one barrier per step publishes them. The first
//     K slice of the next step is read before that barrier, so neither the
//     row loads nor LDS latency sit on the per-step critical path. Only
//     register loads are in flight, so the compiler's load-count waits are
//     exact. (Direct-to-LDS loads mixed with register loads under partial
//     vmcnt waits were observed to read stale LDS data: their completions
//     are not ordered with respect to each other.)
//   * Within a step the instruction order is fixed: MFMAs interleaved with
//     the LDS reads of the next 16-wide K slice and an even share of the
//     step's loads, so a load waiting for queue space never idles the matrix
//     core for long.
//   * A pass covers up to 192 (160) rows of one expert (the accumulators of
//     6 (5) row fragments x 2 column fragments live in AGPRs, one wave per
//     SIMD), so every uniformly routed DeepSeek-V3 expert (128 +- 11 rows) is
//     one pass and its weights are read exactly once, with non-temporal
//     loads. Longer segments take more passes: their fragments are spread
//     evenly over the passes, the passes of one column tile are ordered side
//     by side, and their weight loads are cached, so the passes run together
//     and share the weight stream through L2.
//   * The K loop is compiled per count of active 32-row fragments, so the
//     MFMA stream has no branches.
//   * The expert FFN is one launch (ffn_stream_kernel): every workgroup
//     takes GEMM1 tiles until none is left anywhere, then GEMM2 tiles. A
//     GEMM2 tile first waits until every GEMM1 tile of its group has counted
//     its (complete) stores of h; groups finish in tile-list order, so the
//     wait is rare and short, and the compute units that run out of GEMM1
//     work start on GEMM2 instead of idling until the slowest GEMM1 tile is
//     done. Every tile is claimed from the queues, so a tile that a wait
//     depends on is always held by a running workgroup.
//   * The MFMAs take the weights as their first operand and the token rows
//     as their second, so every lane ends with runs of 4 consecutive output
//     columns of one token row. The epilogue assembles the output tile in
//     LDS and writes it in whole 128-byte lines with streaming stores that
//     bypass L2, so the outputs do not evict the token rows that the column
//     tiles of one expert share through L2.
//
// Packed layout (element = bf16, 8 per 16-byte lane chunk), per expert:
//   GEMM1: [I/128 tiles][K/64 steps][4 waves][4 kk][2 j][64 lanes][8]
//          tile t, wave w owns h columns c = t*128 + w*32 + (lane & 31);
//          j = 0 holds w_gate row c, j = 1 holds w_up row c.
//   GEMM2: [d/256 tiles][I/64 steps][4 waves][4 kk][2 j][64 lanes][8]
//          wave w owns output columns t*256 + w*64 + j*32 + (lane & 31).
//   The 8 elements of (step s, kk, lane) are k = s*64 + kk*16 + 8*(lane>>5) + 0..7.
#include "moe_internal.h"

#include <algorithm>
#include <type_traits>
#include <utility>

namespace moe {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kMaxRows = 192;      // rows per pass
constexpr int kStepBytes = 8192;   // one wave's weights per K step
constexpr int kDepth = 3;          // weight register sets: the current K step and kDepth-1 in flight
constexpr int kSlots = 3;          // A ring slots in LDS: the current step, the next, the one being written
constexpr int kStage = 2;          // A register sets: rows loaded three steps ahead, written two ahead
constexpr int kUnroll = 6;         // K-loop unroll: a multiple of kDepth, kSlots and kStage
constexpr int kStreamStore = 19;   // cache policy of output stores: sc0 sc1 nt (streaming, not kept in L2)
static_assert(kUnroll % kDepth == 0 && kUnroll % kSlots == 0 && kUnroll % kStage == 0, "unroll");

template <bool DEEP>
struct StreamCfg {
  static constexpr int rows = kMaxRows, depth = kDepth, slots = kSlots, unroll = kUnroll;
};
template <>
struct StreamCfg<true> {
  static constexpr int rows = 160, depth = 4, slots = 4, unroll = 4;
};
// Pipeline shapes. The default one keeps two weight steps in flight and
// takes passes of up to 192 rows; the deep one keeps three in flight, which
// fits the register file with passes of up to 160 rows. Deep is measured
// faster for GEMM2 (K = I: short tiles) when the groups are small
// (DeepSeek-V3 shape, ~128 rows per expert); GEMM1 and groups of many
// passes (the Mixtral shape) prefer the default.
constexpr int kDeepMaxAvgRows = 160;

__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
__device__ __forceinline__ void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
__device__ __forceinline__ void barrier_only() { asm volatile("s_barrier" ::: "memory"); }

// A ring layout: 128-byte rows of 8 16-byte chunks, chunk c of row r stored at
// chunk c ^ ((r >> 1) & 7). The 16 rows one quarter-wave reads with a 16-byte
// load (lanes 0-15 or 16-31 of a fragment) then fall on 16 distinct 16-byte
// bank groups.
__device__ __forceinline__ int lds_off(int row, int chunk) { return (row << 7) + ((chunk ^ ((row >> 1) & 7)) << 4); }
__device__ __forceinline__ float silu_f(float g) { return g / (1.0f + __expf(-g)); }

// 16 int8 codes (one 16-byte load, element e in byte e) -> the same 16 values
// as bf16 in two 16-byte chunks (elements 0-7, 8-15). Integers of at most 8
// bits are exact in bf16, so keeping the high half of the fp32 value is exact.
__device__ __forceinline__ void codes_to_bf16(i32x4 v, i32x4& lo, i32x4& hi) {
  uint32_t o[8];
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    float f[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) f[j] = (float)(int)__builtin_amdgcn_sbfe(v[d], 8 * j, 8);  // sign-extended byte j
    // bytes 2,3 of the first value, then bytes 2,3 of the second
    o[2 * d] = __builtin_amdgcn_perm(__float_as_uint(f[1]), __float_as_uint(f[0]), 0x07060302u);
    o[2 * d + 1] = __builtin_amdgcn_perm(__float_as_uint(f[3]), __float_as_uint(f[2]), 0x07060302u);
  }
  lo = i32x4{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
  hi = i32x4{(int)o[4], (int)o[5], (int)o[6], (int)o[7]};
}

// 16 FP8 codes (OCP E4M3, element e in byte e) -> the same 16 values as
// bf16. Every E4M3 value (3 mantissa bits, exponents 2^-9 .. 2^8) is exact
// in bf16, so keeping the high half of the converted fp32 value is exact.
__device__ __forceinline__ void fp8_to_bf16(i32x4 v, i32x4& lo, i32x4& hi) {
  uint32_t o[8];
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    const auto f01 = __builtin_amdgcn_cvt_pk_f32_fp8(v[d], false);  // bytes 0, 1
    const auto f23 = __builtin_amdgcn_cvt_pk_f32_fp8(v[d], true);   // bytes 2, 3
    o[2 * d] = __builtin_amdgcn_perm(__float_as_uint(f01[1]), __float_as_uint(f01[0]), 0x07060302u);
    o[2 * d + 1] = __builtin_amdgcn_perm(__float_as_uint(f23[1]), __float_as_uint(f23[0]), 0x07060302u);
  }
  lo = i32x4{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
  hi = i32x4{(int)o[4], (int)o[5], (int)o[6], (int)o[7]};
}

template <typename F, int... Is>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, Is...>) {
  (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Calls f(std::integral_constant<int, n>) for a runtime n in [LO, N] (n < LO
// runs the LO instance).
template <int N, int LO, typename F>
__device__ __forceinline__ void with_count_from(int n, F&& f) {
  if constexpr (N <= LO) {
    f(std::integral_constant<int, LO>{});
  } else {
    if (n == N) f(std::integral_constant<int, N>{});
    else with_count_from<N - 1, LO>(n, f);
  }
}

__device__ __forceinline__ int scan4(int v, int* scratch, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int n = __shfl_up(inc, o, 64);
    if (lane >= o) inc += n;
  }
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

// Role of one GEMM in a launch: alone, or a phase of the fused FFN launch
// (ffn_stream_kernel): GEMM1 there counts its finished tiles per group
// (PRODUCER), GEMM2 waits for them before reading a group's rows of h
// (CONSUMER). In both phases every tile is claimed from the queues (none is
// implicitly a workgroup's first), so a tile that a wait depends on is always
// held by a running workgroup.
enum { ROLE_ALONE = 0, ROLE_PRODUCER = 1, ROLE_CONSUMER = 2 };
// Polls of a GEMM2 tile's wait (each followed by a short sleep) before it sets
// the wait flag and goes on: about a second, thousands of times any real wait.
constexpr int kWaitPolls = 1 << 22;

// A counter of the fused launch as this moment's value at the coherence
// point: an atomic max with 0 (no change to a non-negative counter). A plain
// load, even an atomic one, may be served from a line that this XCD's L2
// still holds from an earlier read, and a line read that often stays there.
__device__ __forceinline__ int read_counter(int32_t* c) {
  return __hip_atomic_fetch_max(c, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Per-workgroup bookkeeping in static LDS, one copy per launch (the two
// phases of the fused launch use it in turn).
struct StreamLds {
  int tstart[257];            // first tile (pass) of each group
  int scan_scratch[kWaves];
  int next;                   // the workgroup's next tile
  int ready;                  // CONSUMER: every workgroup is done with GEMM1
};

// EPI_SWIGLU: GEMM1 (j = gate/up, 32 output columns per wave);
// EPI_STORE:  GEMM2 (j = two 32-column halves, 64 output columns per wave).
template <int EPI, bool Q8, bool F8, bool DEEP, int ROLE>
__device__ __forceinline__ void stream_gemm(const GemmProblem& p, char* smem, StreamLds& sl) {
  constexpr int kMaxRows = StreamCfg<DEEP>::rows, kDepth = StreamCfg<DEEP>::depth;
  constexpr int kSlots = StreamCfg<DEEP>::slots, kUnroll = StreamCfg<DEEP>::unroll;
  static_assert(kUnroll % kDepth == 0 && kUnroll % kSlots == 0 && kUnroll % kStage == 0, "unroll");
  constexpr int WCOLS = (EPI == EPI_SWIGLU) ? 32 : 64;  // output columns per wave
  constexpr int TCOLS = WCOLS * kWaves;                  // per tile
  // smem (dynamic LDS): the A ring (kSlots slots of kMaxRows x 128 bytes).
  int(&tstart)[257] = sl.tstart;
  int* const scan_scratch = sl.scan_scratch;
  __shared__ float s_scale[kMaxRows];  // Q8: the tile's row scales

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int groups = p.offsets ? p.groups : 1;
  {
    int mt = 0;
    if (tid < groups) {
      int c = p.M;
      if (p.offsets) {
        const int lo = min(max(p.offsets[tid], 0), p.M);
        c = min(max(p.seg_end ? p.seg_end[tid] : p.offsets[tid + 1], lo), p.M) - lo;
      }
      mt = (c + kMaxRows - 1) / kMaxRows;
    }
    int total;
    const int ex = scan4(mt, scan_scratch, &total);
    if (tid < groups) tstart[tid] = ex;
    if (tid == 0) tstart[groups] = total;
    __syncthreads();
  }
  const int Nt = p.N / TCOLS;
  // Work: Nt column tiles per pass (up to kMaxRows rows of one group). The
  // tile sequence is Nt segments: a 1/Nt share of the routed tiles, then the
  // extra group's passes of column tile j side by side (adjacent tiles run on
  // one XCD at the same time and share that weight stream through its L2),
  // so the extra group's compute-heavy full passes run next to memory-heavy
  // routed ones rather than all at the end. GEMM1 of the fused launch puts
  // the passes of two column tiles in each of the first Nt/2 segments, so
  // the extra group's GEMM1 is done by mid-launch and its GEMM2 tiles never
  // wait.
  constexpr int XD = (ROLE == ROLE_PRODUCER) ? 2 : 1;  // column tiles' extra passes per segment
  const int routed_tiles = tstart[groups] * Nt;
  const int units_x = (p.x_rows + kMaxRows - 1) / kMaxRows;
  const int total_tiles = routed_tiles + Nt * units_x;
  auto seg_start = [&](int j) { return (int)((int64_t)j * routed_tiles / Nt) + units_x * min(j * XD, Nt); };
  const int nk = p.K / 64;
  // Rows [row0, row0 + rows) of pass `pass` of a group of c rows taking
  // `passes` passes: the group's 32-row fragments are spread evenly over its
  // passes (at most kMaxRows / 32 each), so the passes of one column tile take
  // about the same time and stay together, sharing the tile's weights in L2.
  auto pass_rows = [&](int c, int passes, int pass, int& row0, int& rows) __attribute__((always_inline)) {
    const int nfrag = (c + 31) / 32;
    const int base = nfrag / passes, rem = nfrag % passes;
    row0 = 32 * (pass * base + min(pass, rem));
    rows = min(32 * (base + (pass < rem ? 1 : 0)), c - row0);
  };
  const int G = gridDim.x, b = blockIdx.x;
  // Schedule. Workgroups are dealt to the 8 XCDs round-robin (b % 8); XCD x
  // owns the queue of tiles {r G + x W + j : j < W} (W = G / 8, r = 0, 1,
  // ...), so adjacent tiles (an expert's column tiles, sharing token rows
  // through L2) run on one XCD. Each workgroup starts with queue entry b / 8
  // and then claims entries W, W + 1, ... from its XCD's queue head; when its
  // queue is empty it takes tiles from the other XCDs' queues. Without queue
  // heads it takes every G-th tile.
  const bool dyn = p.tile_queue != nullptr && G % 8 == 0;  // always, in the fused launch
  const int W = G / 8, xcd = b % 8;
  auto qtile = [&](int x, int q) { return (q / W) * G + x * W + q % W; };
  const int vb = (G % 8 == 0) ? xcd * W + (b / 8) : b;
  constexpr bool CLAIM_ALL = ROLE != ROLE_ALONE;
  const int q0 = CLAIM_ALL ? 0 : W;  // queue entries below q0 are the workgroups' implicit first tiles
  int& s_next = sl.next;
  // this XCD's queue is empty: take a tile from another XCD's queue
  auto steal = [&](int& tile) __attribute__((always_inline)) {
    if (dyn && tile >= total_tiles) {
      __syncthreads();  // every thread has read s_next
      if (tid == 0) {
        int t = total_tiles;
        for (int k = 1; k < 8 && t >= total_tiles; ++k) {
          const int x = (xcd + k) % 8;
          t = qtile(x, q0 + atomicAdd(&p.tile_queue[x], 1));
        }
        s_next = t;
      }
      __syncthreads();
      tile = s_next;
    }
  };
  int tile = vb;
  if constexpr (CLAIM_ALL) {
    if (tid == 0) s_next = qtile(xcd, atomicAdd(&p.tile_queue[xcd], 1));
    __syncthreads();
    tile = s_next;
    steal(tile);
  }
  int pend = -1;  // PRODUCER: group of the previous tile, counted once its stores are complete
  int& s_ready = sl.ready;
  bool ready = false;  // CONSUMER: every workgroup is done with GEMM1 (no tile needs to wait)
  const int K = p.K;
  // A rows move in 1 KB blocks of 8 rows (block b of a wave: rows 32b + 8 wave
  // + 0..7): lane l carries row l/8 of the block and the logical 16-byte chunk
  // that lds_off() places at physical chunk l%8.
  const int lr = lane >> 3, lc = (lane & 7) ^ ((wave * 4 + (lr >> 1)) & 7);
  // Q8: A rows of 1-byte codes (int8, or FP8 with F8) move in 1 KB blocks of 16 rows of 64 bytes
  // (block i of a wave: rows 64 i + 16 wave + 0..15): lane l carries row l/4
  // and codes 16 (l%4) .. 16 (l%4) + 15 of the step's 64.
  const int lr8 = lane >> 2, lc8 = lane & 3;

  while (tile < total_tiles) {
    // claim the next entry of this XCD's queue now; it is used after this tile
    int claim = 0;
    if (dyn && tid == 0) claim = atomicAdd(&p.tile_queue[xcd], 1);
    // ---- decode: group, pass and column tile nt
    int seg = 0;
    if (units_x > 0) {
      int lo = 0, hi = Nt - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (seg_start(mid) <= tile) lo = mid; else hi = mid - 1;
      }
      seg = lo;
    }
    const int r_beg = (int)((int64_t)seg * routed_tiles / Nt);
    const int r_len = (int)((int64_t)(seg + 1) * routed_tiles / Nt) - r_beg;
    const int off = units_x > 0 ? tile - seg_start(seg) : tile;
    const bool extra = units_x > 0 && off >= r_len;  // extra-group tile off - r_len of segment seg
    const void* a_base;
    const int32_t* gather;
    int a_rows, row0, rows, nt;
    const char* b_base;
    __bf16* c_base;
    bool multi;  // the tile's group takes more than one pass
    int gid;     // the tile's group (the extra group: groups)
    if (extra) {
      a_base = p.xA;
      a_rows = p.x_rows;
      gather = nullptr;
      nt = seg * XD + (off - r_len) / units_x;
      gid = groups;
      pass_rows(p.x_rows, units_x, (off - r_len) % units_x, row0, rows);
      multi = units_x > 1;
      b_base = static_cast<const char*>(p.xB) + (size_t)nt * nk * kWaves * kStepBytes;
      c_base = static_cast<__bf16*>(p.xC);
    } else {
      // routed tile rt; an expert's passes of one column tile are side by side
      const int rt = units_x > 0 ? r_beg + off : tile;
      const int q = rt / Nt;
      int lo = 0, hi = groups - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (tstart[mid] <= q) lo = mid; else hi = mid - 1;
      }
      const int e = lo;
      gid = e;
      const int local = rt - tstart[e] * Nt;
      const int passes = tstart[e + 1] - tstart[e];
      const int pass = local % passes;
      multi = passes > 1;
      nt = local / passes;
      const int gbeg = p.offsets ? min(max(p.offsets[e], 0), p.M) : 0;
      const int gend = p.offsets ? min(max(p.seg_end ? p.seg_end[e] : p.offsets[e + 1], gbeg), p.M) : p.M;
      a_base = p.A;
      a_rows = p.a_rows;
      gather = p.gather;
      pass_rows(gend - gbeg, passes, pass, row0, rows);
      row0 += gbeg;
      b_base = static_cast<const char*>(p.B0) + ((size_t)e * Nt + nt) * nk * kWaves * kStepBytes;
      c_base = static_cast<__bf16*>(p.C);
    }
    if constexpr (ROLE == ROLE_CONSUMER) {
      // Wait until every GEMM1 tile of this group (its passes of up to 192
      // rows x its N/128 column tiles, the same rows and count in GEMM1's
      // tile list) has stored its rows of h. Those stores are written
      // through to memory and complete before their count is added. No L2
      // holds an older copy of the rows: the caches start the launch without
      // them and this launch reads them only after the wait, so the loads
      // below see the new values. Once every workgroup is done with GEMM1
      // (the count at groups + 2 reaches the grid), no tile checks again.
      if (!ready) {
        if (tid == 0) {
          int r = read_counter(p.deps + groups + 2) >= G;
          if (!r) {
            int c = p.x_rows;
            if (!extra) {
              const int lo = min(max(p.offsets[gid], 0), p.M);
              c = min(max(p.offsets[gid + 1], lo), p.M) - lo;
            }
            constexpr int kRows1 = StreamCfg<false>::rows, kCols1 = 32 * kWaves;  // GEMM1 pass rows, tile columns
            const int need = (c + kRows1 - 1) / kRows1 * (K / kCols1);
            for (int it = 0; read_counter(p.deps + gid) < need; ++it) {
              if (it == kWaitPolls) {
                __hip_atomic_fetch_or(p.deps + groups + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                break;
              }
              __builtin_amdgcn_s_sleep(8);
            }
          }
          s_ready = r;
        }
        __syncthreads();
        ready = s_ready;
      }
    }
    const __amdgpu_buffer_rsrc_t a_rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<void*>(a_base), (short)0, (int)(uint32_t)((size_t)a_rows * K * (Q8 ? 1 : 2)), 0x00020000);

    // this wave's packed weights: contiguous nk * 32 KB per tile, 8 KB per wave per step
    const char* bw = b_base + (size_t)wave * kStepBytes + lane * 16;

    f32x16 acc[kMaxRows / 32][2];
#pragma unroll
    for (int i = 0; i < kMaxRows / 32; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    const int nact = __builtin_amdgcn_readfirstlane((rows + 31) / 32);

    // TEMPORAL: weight loads that stay in L2 (a pass of a group that takes
    // several passes: the group's other passes of the same column tile run
    // next to it and find its weights there); otherwise non-temporal loads
    // (weights read once).
    auto body = [&](auto ar_c, auto temporal_c) __attribute__((always_inline)) {
      constexpr int AR = decltype(ar_c)::value;  // A rows staged per step (32, 128 or kMaxRows)
      constexpr bool TEMPORAL = decltype(temporal_c)::value;
      constexpr int A_CH = Q8 ? AR / (16 * kWaves) : AR / (8 * kWaves);  // A loads per wave per step
      constexpr int LOADS = A_CH + 8;
      uint32_t a_off[A_CH];  // byte offsets into A (its size is checked below 4 GiB at launch)
#pragma unroll
      for (int i = 0; i < A_CH; ++i) {
        if constexpr (Q8) {
          const int r = min(i * 16 * kWaves + wave * 16 + lr8, rows - 1);
          const int ar = gather ? min(max(gather[row0 + r], 0), a_rows - 1) : row0 + r;
          a_off[i] = (uint32_t)ar * (uint32_t)K + lc8 * 16;
        } else {
          const int r = min(i * 8 * kWaves + wave * 8 + lr, rows - 1);
          const int ar = gather ? min(max(gather[row0 + r], 0), a_rows - 1) : row0 + r;
          a_off[i] = (uint32_t)ar * (uint32_t)(K * 2) + lc * 16;
        }
      }
      // Q8: the scale of tile row tid, written to s_scale before the K loop
      float row_scale = 0.f;
      if constexpr (Q8) {
        if (tid < rows) {
          const int ar = gather ? min(max(gather[row0 + tid], 0), a_rows - 1) : row0 + tid;
          row_scale = p.a_scale[ar];
        }
      }
      // Per wave, in flight: weights for kDepth-1 steps ahead (kDepth register
      // sets) and its share of the A rows of the steps two and three ahead
      // (kStage register sets, written to the LDS ring two steps before use).
      // Every load returns to registers, so the compiler's own wait counts
      // (in-order returns) are exact and no hand-written vmcnt wait is needed.
      i32x4 bq[kDepth][8];
      i32x4 sa[kStage][A_CH];
      // Steps past the end are clamped to the last one: those surplus loads
      // are never used, which keeps the steady-state loop free of branches.
      auto load_a = [&](int ks, auto s_c, int i) __attribute__((always_inline)) {
        const int kc = min(ks, nk - 1);
        sa[decltype(s_c)::value][i] =
            __builtin_amdgcn_raw_buffer_load_b128(a_rs, (int)(a_off[i] + kc * (Q8 ? 64 : 128)), 0, 0);
      };
      auto load_b = [&](int ks, auto s_c, int n) __attribute__((always_inline)) {
        const int kc = min(ks, nk - 1);
        const i32x4* const src = reinterpret_cast<const i32x4*>(bw + (size_t)kc * kWaves * kStepBytes + n * 1024);
        if constexpr (TEMPORAL) bq[decltype(s_c)::value][n] = *src;
        else bq[decltype(s_c)::value][n] = __builtin_nontemporal_load(src);
      };
      // Write A register set S into ring slot R (layout of lds_off(): lane l
      // holds row l/8 of each 8-row block, at physical chunk l%8). Q8: each
      // lane's 16 codes become the row's bf16 chunks 2 (l%4) and 2 (l%4) + 1.
      auto stage = [&](auto s_c, auto r_c) __attribute__((always_inline)) {
        if constexpr (Q8) {
          char* const slot = smem + decltype(r_c)::value * (kMaxRows * 128);
#pragma unroll
          for (int i = 0; i < A_CH; ++i) {
            const int r = i * 16 * kWaves + wave * 16 + lr8;
            i32x4 lo, hi;
            if constexpr (F8) fp8_to_bf16(sa[decltype(s_c)::value][i], lo, hi);
            else codes_to_bf16(sa[decltype(s_c)::value][i], lo, hi);
            *reinterpret_cast<i32x4*>(slot + lds_off(r, 2 * lc8)) = lo;
            *reinterpret_cast<i32x4*>(slot + lds_off(r, 2 * lc8 + 1)) = hi;
          }
        } else {
          char* const dst = smem + decltype(r_c)::value * (kMaxRows * 128) + wave * 8 * 128 + lane * 16;
#pragma unroll
          for (int i = 0; i < A_CH; ++i)
            *reinterpret_cast<i32x4*>(dst + i * 8 * kWaves * 128) = sa[decltype(s_c)::value][i];
        }
      };

      auto kloop = [&](auto nact_c) __attribute__((always_inline)) {
        constexpr int NACT = decltype(nact_c)::value;
        auto rd = [&](int slot, int kk, int i) __attribute__((always_inline)) {
          return *reinterpret_cast<const i32x4*>(smem + slot * (kMaxRows * 128) +
                                                 lds_off(32 * i + (lane & 31), 2 * kk + (lane >> 5)));
        };
        i32x4 af[NACT > 0 ? NACT : 1];  // A fragments of the current 16-wide K slice
        // Step ks (U = ks % kUnroll) multiplies slot U % kSlots with weight set
        // U % kDepth while loading step ks+3's A rows and step ks+kDepth-1's
        // weights. At its end it writes step ks+2's A rows into slot
        // (U+2) % kSlots (last read by step ks-1, which every wave finished
        // before the previous barrier), reads the first K slice of step ks+1
        // (published by the previous barrier) and meets the others at a
        // barrier, so no LDS latency sits between the barrier and the MFMAs.
        // TAIL: one of the last steps, whose loads past the last K step are
        // skipped (elsewhere every load is in range, and the loads stay
        // unconditional so the compiler's wait counts are exact).
        auto step = [&](int ks, auto u_c, auto tail_c) __attribute__((always_inline)) {
          constexpr int U = decltype(u_c)::value;
          constexpr bool TAIL = decltype(tail_c)::value;
          const bool a_ok = !TAIL || ks + 3 < nk, b_ok = !TAIL || ks + kDepth - 1 < nk;
          constexpr int SL = U % kSlots, BS = U % kDepth;
          constexpr auto SB = std::integral_constant<int, (U + kDepth - 1) % kDepth>{};
          constexpr auto SA3 = std::integral_constant<int, (U + 3) % kStage>{};  // set of step ks+3
          constexpr auto SA2 = std::integral_constant<int, (U + 2) % kStage>{};  // set of step ks+2
          constexpr auto SL2 = std::integral_constant<int, (U + 2) % kSlots>{};
          __builtin_amdgcn_sched_barrier(0);
          if constexpr (NACT > 0) {
            // Fixed instruction order (each group closed by a scheduling
            // barrier): per row fragment the two MFMAs of one slice, the read
            // of the same fragment's next slice (NACT groups to land) and an
            // even share of this step's loads (A rows first). Spreading the
            // loads keeps a load that waits for queue space from idling the
            // matrix core for long.
            constexpr int GROUPS = 4 * NACT;
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
#pragma unroll
              for (int i = 0; i < NACT; ++i) {
                const int g = kk * NACT + i;
#pragma unroll
                for (int j = 0; j < 2; ++j)
                  acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, bq[BS][kk * 2 + j]),
                                                                      __builtin_bit_cast(bf16x8, af[i]),
                                                                      acc[i][j], 0, 0, 0);
                if (kk < 3) af[i] = rd(SL, kk + 1, i);
#pragma unroll
                for (int n = g * LOADS / GROUPS; n < (g + 1) * LOADS / GROUPS; ++n) {
                  if (n < A_CH) {
                    if (a_ok) load_a(ks + 3, SA3, n);
                  } else if (b_ok) {
                    load_b(ks + kDepth - 1, SB, n - A_CH);
                  }
                }
                __builtin_amdgcn_sched_barrier(0);
              }
            }
          } else {
#pragma unroll
            for (int i = 0; i < A_CH; ++i)
              if (a_ok) load_a(ks + 3, SA3, i);
#pragma unroll
            for (int n = 0; n < 8; ++n)
              if (b_ok) load_b(ks + kDepth - 1, SB, n);
          }
          stage(SA2, SL2);
          lds_wait();  // this wave's ring writes (and reads) are done
#pragma unroll
          for (int i = 0; i < NACT; ++i) af[i] = rd((U + 1) % kSlots, 0, i);
          barrier_only();
        };
        lds_barrier();  // every wave is done with the previous tile's ring
        static_for<kStage>([&](auto s_c) {
#pragma unroll
          for (int i = 0; i < A_CH; ++i) load_a(decltype(s_c)::value, s_c, i);
        });
        static_for<kDepth - 1>([&](auto s_c) {
#pragma unroll
          for (int n = 0; n < 8; ++n) load_b(decltype(s_c)::value, s_c, n);
        });
        stage(std::integral_constant<int, 0>{}, std::integral_constant<int, 0>{});
        stage(std::integral_constant<int, 1>{}, std::integral_constant<int, 1>{});
        if constexpr (Q8) {
          if (tid < kMaxRows) s_scale[tid] = row_scale;  // published by the barrier below
        }
        // step 2's rows take set 0 (free again); step 0 then loads step 3's
#pragma unroll
        for (int i = 0; i < A_CH; ++i) load_a(2, std::integral_constant<int, 0>{}, i);
        lds_barrier();  // slots 0 and 1 written by every wave
#pragma unroll
        for (int i = 0; i < NACT; ++i) af[i] = rd(0, 0, i);
        int ks = 0;
        // main loop: every load of its steps is in range (ks + kUnroll + 2 < nk)
        for (; ks + kUnroll + 2 < nk; ks += kUnroll)
          static_for<kUnroll>([&](auto u_c) { step(ks + u_c, u_c, std::false_type{}); });
        static_for<kUnroll + 2>([&](auto u_c) {
          if (ks + u_c < nk) step(ks + u_c, std::integral_constant<int, decltype(u_c)::value % kUnroll>{}, std::true_type{});
        });
      };
      // A pass of more than 128 rows has at least 5 fragments; with the
      // fragments spread evenly, every pass of a group that takes several
      // passes has at least 3.
      with_count_from<AR / 32, (AR > 128 ? 5 : (TEMPORAL ? 3 : 0))>(min(nact, AR / 32), kloop);
    };
    // A single pass of at most 32 rows stages one 32-row fragment: one token-row
    // load per wave and step instead of four copies of its last row
    // (bf16 tokens; a 32-row block of 1-byte codes would be half a load).
    bool thin = false;
    if constexpr (!Q8) {
      if (rows <= 32 && !multi) {
        body(std::integral_constant<int, 32>{}, std::false_type{});
        thin = true;
      }
    }
    if (thin) {
    } else if (rows <= 128) {
      if (multi) body(std::integral_constant<int, 128>{}, std::true_type{});
      else body(std::integral_constant<int, 128>{}, std::false_type{});
    } else if (multi) body(std::integral_constant<int, kMaxRows>{}, std::true_type{});
    else body(std::integral_constant<int, kMaxRows>{}, std::false_type{});

    // ---- epilogue. The MFMAs take the weights as their first operand, so
    // acc[i][j] is the transposed 32x32 tile: lane l holds token row
    // 32 i + l%32 and output columns 32 j + 8 g + 4 (l/32) + 0..3 in
    // registers 4 g .. 4 g + 3. Those 8-byte runs go into an LDS copy of the
    // output tile (rows x TCOLS bf16, 16-byte chunks XOR-swizzled by row);
    // the tile then leaves in whole 128-byte lines, one 16-byte chunk per
    // thread per pass, OROWS rows per pass, as streaming stores that bypass
    // L2 (written once, read by a later kernel): write-allocated output
    // lines would evict the token rows the column tiles share through L2.
    {
      constexpr int OCH = TCOLS * 2 / 16;      // 16-byte chunks per output row
      constexpr int OROWS = kThreads / OCH;    // rows per store pass
      if (tid == 0) s_next = dyn ? qtile(xcd, q0 + claim) : tile + G;
      // PRODUCER: the previous tile's stores (issued a whole tile ago) are
      // complete; no load is in flight at this point (the K loop's last
      // steps skip every load past the last step)
      if constexpr (ROLE == ROLE_PRODUCER) {
        if (pend >= 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      }
      lds_barrier();                           // every wave is done reading the A ring
      if constexpr (ROLE == ROLE_PRODUCER) {
        if (pend >= 0 && tid == 0) __hip_atomic_fetch_add(p.deps + pend, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        pend = gid;
      }
      const int h = lane >> 5;
#pragma unroll
      for (int i = 0; i < kMaxRows / 32; ++i) {
        __builtin_amdgcn_sched_barrier(0);  // one fragment at a time: few live registers
        if (i < nact) {
          const int r = 32 * i + (lane & 31);
          char* const orow = smem + r * (TCOLS * 2);
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            if (EPI == EPI_SWIGLU) {
              bf16x4 v;
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                // Q8: the sums ran over the codes; the row's scale restores the tokens
                const float sc = Q8 ? s_scale[r] : 1.0f;
                v[e] = static_cast<__bf16>(silu_f(acc[i][0][4 * g + e] * sc) * (acc[i][1][4 * g + e] * sc));
              }
              const int c = wave * 4 + g;
              *reinterpret_cast<bf16x4*>(orow + ((c ^ (r & 7)) << 4) + 8 * h) = v;
            } else {
#pragma unroll
              for (int j = 0; j < 2; ++j) {
                bf16x4 v;
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = static_cast<__bf16>(acc[i][j][4 * g + e]);
                const int c = wave * 8 + 4 * j + g;
                *reinterpret_cast<bf16x4*>(orow + ((c ^ (r & 7)) << 4) + 8 * h) = v;
              }
            }
          }
        }
      }
      lds_barrier();
      const size_t ldc = (size_t)p.ldc;
      char* const cb = reinterpret_cast<char*>(c_base) + ((size_t)row0 * ldc + (size_t)nt * TCOLS) * 2;
      // rows >= `rows` fall outside the buffer range: the hardware drops them
      const __amdgpu_buffer_rsrc_t c_rs =
          __builtin_amdgcn_make_buffer_rsrc(cb, (short)0, (int)((uint32_t)rows * (uint32_t)(ldc * 2)), 0x00020000);
      const int oc = tid % OCH;
      const int npass = (rows + OROWS - 1) / OROWS;
#pragma unroll
      for (int q = 0; q < kMaxRows / OROWS; ++q) {
        if (q % 4 == 0) __builtin_amdgcn_sched_barrier(0);  // a few rows in flight: few live registers
        if (q < npass) {
          const int r = q * OROWS + tid / OCH;
          const i32x4 v = *reinterpret_cast<const i32x4*>(smem + r * (TCOLS * 2) + ((oc ^ (r & 7)) << 4));
          __builtin_amdgcn_raw_buffer_store_b128(v, c_rs, (int)((uint32_t)r * (uint32_t)(ldc * 2) + oc * 16), 0,
                                                 kStreamStore);
        }
      }
    }
    tile = s_next;  // written before the epilogue's barriers
    steal(tile);
  }
  if constexpr (ROLE == ROLE_PRODUCER) {
    // the last tile's count, once every thread's stores are complete, then
    // (after that count is performed) this workgroup's end of GEMM1
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (tid == 0) {
      if (pend >= 0) __hip_atomic_fetch_add(p.deps + pend, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __hip_atomic_fetch_add(p.deps + groups + 2, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();  // the LDS and s_next are free for the next phase
  }
}

template <int EPI, bool Q8, bool F8, bool DEEP>
__global__ void __launch_bounds__(kThreads, 1) gemm_stream_kernel(GemmProblem p) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ StreamLds sl;
  stream_gemm<EPI, Q8, F8, DEEP, ROLE_ALONE>(p, smem, sl);
}

// The expert FFN in one launch: GEMM1+SwiGLU over bf16 tokens, then GEMM2
// (DEEP2: its deep pipeline shape) on the same workgroups, so the end of
// GEMM1 overlaps the start of GEMM2 instead of idling compute units.
template <bool DEEP2>
__global__ void __launch_bounds__(kThreads, 1) ffn_stream_kernel(GemmProblem up, GemmProblem down) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ StreamLds sl;
  stream_gemm<EPI_SWIGLU, false, false, false, ROLE_PRODUCER>(up, smem, sl);
  stream_gemm<EPI_STORE, false, false, DEEP2, ROLE_CONSUMER>(down, smem, sl);
}

__global__ void queue_reset_kernel(int32_t* q, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) q[i] = 0;
}

// One 16-byte chunk per thread: packed position -> source row and k.
__global__ void pack_kernel(const __bf16* __restrict__ w0, const __bf16* __restrict__ w1, __bf16* __restrict__ dst,
                            int E, int N, int K, int gate_up) {
  const int tcols = gate_up ? 128 : 256;
  const int nt_all = N / tcols, nk = K / 64;
  const size_t chunks_per_expert = (size_t)N * K / 8 * (gate_up ? 2 : 1);
  const size_t total = chunks_per_expert * E;
  for (size_t c = (size_t)blockIdx.x * blockDim.x + threadIdx.x; c < total; c += (size_t)gridDim.x * blockDim.x) {
    size_t r = c;
    const int lane = (int)(r % 64); r /= 64;
    const int j = (int)(r % 2); r /= 2;
    const int kk = (int)(r % 4); r /= 4;
    const int w = (int)(r % 4); r /= 4;
    const int s = (int)(r % nk); r /= nk;
    const int nt = (int)(r % nt_all); r /= nt_all;
    const int e = (int)r;
    const int k0 = s * 64 + kk * 16 + 8 * (lane >> 5);
    const __bf16* src;
    int row;
    if (gate_up) {
      row = nt * 128 + w * 32 + (lane & 31);
      src = j ? w1 : w0;
    } else {
      row = nt * 256 + w * 64 + j * 32 + (lane & 31);
      src = w0;
    }
    const i32x4 v = *reinterpret_cast<const i32x4*>(src + ((size_t)e * N + row) * K + k0);
    *reinterpret_cast<i32x4*>(dst + c * 8) = v;
  }
}

template <int EPI, bool Q8, bool F8 = false, bool DEEP = false>
hipError_t launch_stream(const GemmProblem& p, hipStream_t s) {
  auto kern = gemm_stream_kernel<EPI, Q8, F8, DEEP>;
  // the A ring, reused after each tile's K loop as the LDS copy of its output
  constexpr int kMaxRows = StreamCfg<DEEP>::rows, kSlots = StreamCfg<DEEP>::slots;
  constexpr size_t lds = std::max<size_t>((size_t)kSlots * kMaxRows * 128,
                                          (size_t)kMaxRows * ((EPI == EPI_SWIGLU) ? 128 : 256) * 2);
  const hipError_t init_err = set_dynamic_lds((const void*)kern, (int)lds);
  if (init_err != hipSuccess) return init_err;
  // A is addressed through a buffer resource: 32-bit byte offsets.
  if ((size_t)p.a_rows * (size_t)p.K * (Q8 ? 1 : 2) > 0xFFFFFFFFull || (size_t)p.x_rows * (size_t)p.K * 2 > 0xFFFFFFFFull)
    return hipErrorInvalidValue;
  if (Q8 && (p.x_rows != 0 || !p.a_scale)) return hipErrorInvalidValue;
  if (p.x_rows < 0 || (p.x_rows > 0 && (!p.xA || !p.xB || !p.xC))) return hipErrorInvalidValue;
  const int tcols = (EPI == EPI_SWIGLU) ? 128 : 256;
  const int groups = p.offsets ? p.groups : 1;
  const long long passes_upper =
      (p.M + kMaxRows - 1) / kMaxRows + (p.offsets ? groups : 0) + (p.x_rows + kMaxRows - 1) / kMaxRows;
  const long long upper = passes_upper * (p.N / tcols);
  if (upper <= 0) return hipSuccess;
  long long grid = device_cu_count();
  if (p.max_wg > 0 && grid > p.max_wg) grid = p.max_wg;
  if (grid > upper) grid = upper;
  if (grid >= 8) grid -= grid % 8;
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kThreads), lds, s, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_stream(const GemmProblem& p, int epi, hipStream_t s) {
  if ((p.M <= 0 && p.x_rows <= 0) || p.N <= 0) return hipSuccess;
  // groups of many rows are bound by the matrix cores, not by the weight stream
  if (gemm_dense_eligible(p)) return launch_gemm_dense(p, epi, s);
  if (p.a_scale) {
    if (epi != EPI_SWIGLU) return hipErrorInvalidValue;
    return p.a_fp8 ? launch_stream<EPI_SWIGLU, true, true>(p, s) : launch_stream<EPI_SWIGLU, true>(p, s);
  }
  const int groups = p.offsets ? p.groups : 1;
  const bool small = groups > 0 && (long long)p.M <= (long long)kDeepMaxAvgRows * groups;
  if (epi == EPI_SWIGLU) return launch_stream<EPI_SWIGLU, false>(p, s);
  if (small) return launch_stream<EPI_STORE, false, false, true>(p, s);
  return launch_stream<EPI_STORE, false>(p, s);
}

hipError_t launch_queue_reset(int32_t* q, int n, hipStream_t s) {
  if (!q || n <= 0 || n > 4096) return hipErrorInvalidValue;
  hipLaunchKernelGGL(queue_reset_kernel, dim3(1), dim3(256), 0, s, q, n);
  return hipGetLastError();
}

namespace {

template <bool DEEP2>
hipError_t launch_ffn(const GemmProblem& up, const GemmProblem& down, long long grid, hipStream_t s) {
  auto kern = ffn_stream_kernel<DEEP2>;
  // the larger of the two phases' LDS (each phase's ring, reused as its output tile)
  constexpr size_t lds1 = std::max<size_t>((size_t)StreamCfg<false>::slots * StreamCfg<false>::rows * 128,
                                           (size_t)StreamCfg<false>::rows * 128 * 2);
  constexpr size_t lds2 = std::max<size_t>((size_t)StreamCfg<DEEP2>::slots * StreamCfg<DEEP2>::rows * 128,
                                           (size_t)StreamCfg<DEEP2>::rows * 256 * 2);
  constexpr size_t lds = std::max(lds1, lds2);
  const hipError_t init_err = set_dynamic_lds((const void*)kern, (int)lds);
  if (init_err != hipSuccess) return init_err;
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kThreads), lds, s, up, down);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_ffn_stream(const GemmProblem& up, const GemmProblem& down, hipStream_t s) {
  // bf16 tokens, whole groups of a dispatch, the compute units to itself,
  // and a weight-streaming problem in both GEMMs (nothing is launched when
  // it does not fit: the caller then makes the two launches)
  if (!up.deps || up.deps != down.deps || !up.tile_queue || !down.tile_queue || !up.offsets ||
      up.offsets != down.offsets || up.groups != down.groups || up.groups < 1 || up.groups > kFfnDepsInts - 3)
    return hipErrorNotSupported;
  if (up.a_scale || up.seg_end || down.seg_end || up.max_wg || down.max_wg || up.x_rows != down.x_rows ||
      up.N != down.K || up.M != down.M)
    return hipErrorNotSupported;
  if (gemm_dense_eligible(up) || gemm_dense_eligible(down)) return hipErrorNotSupported;
  if (up.N % 128 != 0 || down.N % 256 != 0 || up.K % 64 != 0 || down.K % 64 != 0) return hipErrorInvalidValue;
  // A is addressed through buffer resources: 32-bit byte offsets
  if ((size_t)up.a_rows * (size_t)up.K * 2 > 0xFFFFFFFFull || (size_t)up.x_rows * (size_t)up.K * 2 > 0xFFFFFFFFull ||
      (size_t)down.a_rows * (size_t)down.K * 2 > 0xFFFFFFFFull ||
      (size_t)down.x_rows * (size_t)down.K * 2 > 0xFFFFFFFFull)
    return hipErrorInvalidValue;
  if (up.x_rows < 0 || (up.x_rows > 0 && (!up.xA || !up.xB || !up.xC || !down.xA || !down.xB || !down.xC)))
    return hipErrorInvalidValue;
  const bool small = (long long)down.M <= (long long)kDeepMaxAvgRows * down.groups;
  const int rows1 = StreamCfg<false>::rows, rows2 = small ? StreamCfg<true>::rows : StreamCfg<false>::rows;
  const long long upper1 = ((up.M + rows1 - 1) / rows1 + up.groups + (up.x_rows + rows1 - 1) / rows1) * (up.N / 128);
  const long long upper2 =
      ((down.M + rows2 - 1) / rows2 + down.groups + (down.x_rows + rows2 - 1) / rows2) * (down.N / 256);
  long long grid = std::min<long long>(device_cu_count(), std::max(upper1, upper2));
  grid -= grid % 8;
  if (grid < 8) return hipErrorNotSupported;  // the tile queues need a multiple of 8 workgroups
  return small ? launch_ffn<true>(up, down, grid, s) : launch_ffn<false>(up, down, grid, s);
}

hipError_t launch_pack(const void* w0, const void* w1, void* dst, int E, int N, int K, bool gate_up, hipStream_t s) {
  const size_t chunks = (size_t)E * N * K / 8 * (gate_up ? 2 : 1);
  if (chunks == 0) return hipSuccess;
  const unsigned grid = (unsigned)std::min<size_t>((chunks + 255) / 256, (size_t)device_cu_count() * 16);
  hipLaunchKernelGGL(pack_kernel, dim3(grid), dim3(256), 0, s, static_cast<const __bf16*>(w0),
                     static_cast<const __bf16*>(w1), static_cast<__bf16*>(dst), E, N, K, gate_up ? 1 : 0);
  return hipGetLastError();
}

}  // namespace moe
