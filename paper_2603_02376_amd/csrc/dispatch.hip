// Dispatch: the single-GPU form of the paper's dispatch all-to-all (App. F,
// first exchange; App. M, variable-size unpadded per-destination transfers).
//
// The T*k assignments (t, j) -> expert topk_idx[t][j] are grouped by expert,
// tokens ascending inside every group: a stable counting sort. Stability is
// what makes the permutation a well-defined, bit-reproducible result, so no
// atomic may decide the order of rows. Three small kernels:
//
//   1. count   — one wavefront per chunk of 64 tokens; lane = token. Every lane
//                ORs its bit into an LDS bitmask per expert it selected (a
//                token holds at most one slot per expert). The masks are
//                written out per (chunk, expert). OR is order-independent, so
//                the masks are deterministic.
//   2. scan    — one workgroup: per expert, the exclusive prefix of popcounts
//                over chunks (the chunk's base inside the expert's segment),
//                the per-expert count, and the exclusive prefix over experts
//                (offsets); optionally it also zeroes the expert GEMMs'
//                tile-queue heads.
//   3. scatter — same grid as 1: the row of (t, j) is
//                offsets[e] + base[chunk][e] + popcount(mask[chunk][e] & lanes below t),
//                i.e. the number of earlier tokens that chose e.
#include "moe_internal.h"

#include <mutex>

// Scratch of moe_dispatch_noalloc: the per-chunk masks and bases of a
// dispatch whose caller passes no workspace. One copy per GPU, held until
// the process ends. In host code this name is only a stand-in for the
// symbol: the device address comes from hipGetSymbolAddress (per device).
static __device__ __align__(256) unsigned char scratch[moe::kDispatchNoAllocBytes];

namespace moe {
namespace {

constexpr int kWaves = 4;  // chunks per workgroup

// A token's expert choices are read kSlotBatch at a time with unconditional
// loads (slot indices clamped to k - 1; the caller drops slots >= k), so the
// loads of a batch are in flight together rather than one after another.
constexpr int kSlotBatch = 8;

__device__ __forceinline__ void load_slots(const DispatchParams& p, int t, int jb, int (&ev)[kSlotBatch]) {
#pragma unroll
  for (int j = 0; j < kSlotBatch; ++j) ev[j] = p.topk_idx[(size_t)t * p.k + min(jb + j, p.k - 1)];
}

__global__ void __launch_bounds__(64 * kWaves) dispatch_count_kernel(DispatchParams p) {
  __shared__ unsigned long long m[kWaves][256];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nchunks = (p.T + kDispatchChunk - 1) / kDispatchChunk;
  const int chunk = blockIdx.x * kWaves + wave;
  const int t = chunk * kDispatchChunk + lane;
  for (int e = lane; e < p.E; e += 64) m[wave][e] = 0ull;
  __syncthreads();
  if (chunk < nchunks && t < p.T) {
    for (int jb = 0; jb < p.k; jb += kSlotBatch) {
      int ev[kSlotBatch];
      load_slots(p, t, jb, ev);
#pragma unroll
      for (int j = 0; j < kSlotBatch; ++j)
        if (jb + j < p.k && (unsigned)ev[j] < (unsigned)p.E) atomicOr(&m[wave][ev[j]], 1ull << lane);
    }
  }
  __syncthreads();
  if (chunk < nchunks)
    for (int e = lane; e < p.E; e += 64) p.masks[(size_t)chunk * p.E + e] = m[wave][e];
}

// One workgroup of 1024 threads: thread (part, e) with part in [0, 4) scans a
// quarter of the chunks for expert e; the four partial sums are combined
// through LDS. Masks are read in batches of kScanBatch chunks whose loads are
// unconditional (indices clamped into the thread's range, popcounts past it
// dropped), so a batch's loads are all in flight together. Up to one batch
// per thread (T <= 4096 tokens) the popcounts stay in registers for the
// second pass; beyond that the second pass reads the masks again.
constexpr int kScanBatch = 16;

__device__ __forceinline__ void scan_batch(const DispatchParams& p, int e, int cb, int c1, int (&pc)[kScanBatch]) {
  unsigned long long m[kScanBatch];
#pragma unroll
  for (int i = 0; i < kScanBatch; ++i) m[i] = p.masks[(size_t)min(cb + i, c1 - 1) * p.E + e];
#pragma unroll
  for (int i = 0; i < kScanBatch; ++i) pc[i] = (cb + i < c1) ? __popcll(m[i]) : 0;
}

__global__ void __launch_bounds__(1024) dispatch_scan_kernel(DispatchParams p) {
  __shared__ int part_sum[4][256];
  __shared__ int wsum[16];
  const int e = threadIdx.x & 255;
  const int part = threadIdx.x >> 8;
  if (p.zero && (int)threadIdx.x < p.n_zero) p.zero[threadIdx.x] = 0;
  const int nchunks = (p.T + kDispatchChunk - 1) / kDispatchChunk;
  const int per = (nchunks + 3) / 4;
  const int c0 = part * per, c1 = min(nchunks, c0 + per);
  const bool active = e < p.E && c0 < c1;  // c1 - 1 is then a valid chunk
  const bool regs = per <= kScanBatch;
  int pc[kScanBatch];
  int run = 0;
  if (active) {
    for (int cb = c0; cb < c1; cb += kScanBatch) {
      scan_batch(p, e, cb, c1, pc);
#pragma unroll
      for (int i = 0; i < kScanBatch; ++i) run += pc[i];
    }
  }
  part_sum[part][e] = run;
  __syncthreads();
  int base = 0, cnt = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int v = part_sum[q][e];
    if (q < part) base += v;
    cnt += v;
  }
  if (active) {
    for (int cb = c0; cb < c1; cb += kScanBatch) {
      if (!regs) scan_batch(p, e, cb, c1, pc);  // one batch: pc still holds it
#pragma unroll
      for (int i = 0; i < kScanBatch; ++i) {
        if (cb + i < c1) {
          p.bases[(size_t)(cb + i) * p.E + e] = base;
          base += pc[i];
        }
      }
    }
  }
  // exclusive scan of the counts over experts (threads of part 0)
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int v = (part == 0 && e < p.E) ? cnt : 0;
  int inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int n = __shfl_up(inc, o, 64);
    if (lane >= o) inc += n;
  }
  if (lane == 63) wsum[wave] = inc;
  __syncthreads();
  if (part == 0) {
    int off = 0, tot = 0;
    for (int w = 0; w < 4; ++w) {
      if (w < wave) off += wsum[w];
      tot += wsum[w];
    }
    if (e < p.E) {
      p.counts[e] = cnt;
      p.offsets[e] = off + inc - v;
    }
    if (e == 0) p.offsets[p.E] = tot;
  }
}

__global__ void __launch_bounds__(64 * kWaves) dispatch_scatter_kernel(DispatchParams p) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int chunk = blockIdx.x * kWaves + wave;
  const int t = chunk * kDispatchChunk + lane;
  if (t >= p.T) return;
  const unsigned long long below = (1ull << lane) - 1ull;
  for (int jb = 0; jb < p.k; jb += kSlotBatch) {
    int ev[kSlotBatch], off[kSlotBatch], base[kSlotBatch];
    unsigned long long mk[kSlotBatch];
    load_slots(p, t, jb, ev);
#pragma unroll
    for (int j = 0; j < kSlotBatch; ++j) {  // every load of the batch issued before any use
      const int ec = min(max(ev[j], 0), p.E - 1);
      const size_t ci = (size_t)chunk * p.E + ec;
      off[j] = p.offsets[ec];
      base[j] = p.bases[ci];
      mk[j] = p.masks[ci];
    }
#pragma unroll
    for (int j = 0; j < kSlotBatch; ++j) {
      // slots past k, and invalid expert ids (row left unassigned), are dropped
      if (jb + j >= p.k || (unsigned)ev[j] >= (unsigned)p.E) continue;
      const int a = t * p.k + jb + j;
      const int row = off[j] + base[j] + __popcll(mk[j] & below);
      p.sorted_token[row] = t;
      if (p.sorted_assign) p.sorted_assign[row] = a;
      p.inv_perm[a] = row;
    }
  }
}

}  // namespace

hipError_t dispatch_noalloc_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  static std::mutex mu;
  static void* addr[64] = {};
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* a = nullptr;
    if ((e = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch))) != hipSuccess) return e;
    if (!a) return hipErrorInvalidSymbol;
    addr[dev] = a;
  }
  *out = addr[dev];
  return hipSuccess;
}

hipError_t launch_dispatch(const DispatchParams& p, hipStream_t s) {
  const int nchunks = (p.T + kDispatchChunk - 1) / kDispatchChunk;
  const int blocks = (nchunks + kWaves - 1) / kWaves;
  if (blocks > 0) hipLaunchKernelGGL(dispatch_count_kernel, dim3(blocks), dim3(64 * kWaves), 0, s, p);
  hipLaunchKernelGGL(dispatch_scan_kernel, dim3(1), dim3(1024), 0, s, p);
  if (blocks > 0) hipLaunchKernelGGL(dispatch_scatter_kernel, dim3(blocks), dim3(64 * kWaves), 0, s, p);
  return hipGetLastError();
}

}  // namespace moe
