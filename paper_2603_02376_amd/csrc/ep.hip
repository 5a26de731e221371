// Row movement on the receive side of expert parallelism (one GPU's share).
//
// In the paper's MoE workload (App. M, §4.3) every GPU owns a subset of the
// experts; the dispatch exchange brings each GPU the token rows routed to its
// experts: its own tokens' rows ("self", available at once) and the peers'
// rows ("remote", available when the exchange has delivered them). The
// receive buffer holds one row per (token, local expert) assignment, grouped
// by expert; within expert e the self rows come first:
//   rows [offsets[e], self_end[e])       self rows,   x_self[row_token[r]]
//   rows [self_end[e], offsets[e + 1])   remote rows, x_peer[row_token[r]]
// This kernel fills the self or the remote rows of an expert range. Run with
// few workgroups on its own stream it stands in for the exchange link: its
// rate is set by the workgroups it may use, and the expert GEMMs on the
// other stream keep the remaining compute units.
#include "moe_internal.h"

namespace moe {
namespace {

constexpr int kThreads = 256;

__global__ void __launch_bounds__(kThreads) ep_copy_kernel(EpCopyParams p) {
  __shared__ int s_off[257];
  __shared__ int s_end[256];
  const int ne = p.e1 - p.e0;  // 1 .. 256, checked at launch
  for (int i = threadIdx.x; i <= ne; i += kThreads) s_off[i] = min(max(p.offsets[p.e0 + i], 0), p.n_rows);
  __syncthreads();
  for (int i = threadIdx.x; i < ne; i += kThreads) s_end[i] = min(max(p.self_end[p.e0 + i], s_off[i]), p.n_rows);
  __syncthreads();
  const int r0 = s_off[0], r1 = max(s_off[ne], r0);
  const int chunks = p.row_bytes / 16;
  for (int r = r0 + (int)blockIdx.x; r < r1; r += (int)gridDim.x) {
    // expert of row r: the last e with s_off[e] <= r (malformed offsets give
    // some e in range: unspecified rows, never an access out of bounds)
    int lo = 0, hi = ne - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s_off[mid] <= r) lo = mid; else hi = mid - 1;
    }
    const bool remote = r >= s_end[lo];
    if (remote != (p.mode == 1)) continue;
    const int t = min(max(p.row_token[r], 0), p.src_rows - 1);
    const i32x4* src = reinterpret_cast<const i32x4*>(static_cast<const char*>(p.src) + (size_t)t * p.row_bytes);
    i32x4* dst = reinterpret_cast<i32x4*>(static_cast<char*>(p.dst) + (size_t)r * p.row_bytes);
    for (int c = threadIdx.x; c < chunks; c += kThreads) dst[c] = __builtin_nontemporal_load(src + c);
  }
}

// One workgroup per local expert e (global expert e_first + e): its rows in
// the receive buffer are this GPU's dispatched rows of that expert, then the
// peer's, each in the order of its dispatch (token ascending).
__global__ void __launch_bounds__(kThreads) ep_plan_kernel(EpPlanParams p) {
  const int e = blockIdx.x, g = p.e_first + e;
  auto so = [&](int i) { return min(max(p.self_offsets[i], 0), p.self_total); };
  auto po = [&](int i) { return min(max(p.peer_offsets[i], 0), p.peer_total); };
  const int s_lo = so(g), s_n = max(so(g + 1) - s_lo, 0);
  const int p_lo = po(g), p_n = max(po(g + 1) - p_lo, 0);
  const int base = max(s_lo - so(p.e_first), 0) + max(p_lo - po(p.e_first), 0);
  if (threadIdx.x == 0) {
    p.offsets[e] = base;
    p.self_end[e] = base + s_n;
    if (e == p.e_count - 1) p.offsets[e + 1] = base + s_n + p_n;
  }
  for (int i = threadIdx.x; i < s_n; i += kThreads)
    if (base + i < p.capacity) p.row_token[base + i] = p.self_sorted[s_lo + i];
  for (int i = threadIdx.x; i < p_n; i += kThreads)
    if (base + s_n + i < p.capacity) p.row_token[base + s_n + i] = p.peer_sorted[p_lo + i];
}

}  // namespace

hipError_t launch_ep_plan(const EpPlanParams& p, hipStream_t s) {
  if (p.e_count <= 0) return hipSuccess;
  if (p.e_first < 0 || p.self_total < 0 || p.peer_total < 0 || p.capacity < 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(ep_plan_kernel, dim3((unsigned)p.e_count), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_ep_copy(const EpCopyParams& p, int max_wg, hipStream_t s) {
  if (p.e1 <= p.e0 || p.n_rows <= 0) return hipSuccess;
  if (p.e0 < 0 || p.e1 - p.e0 > 256 || p.row_bytes <= 0 || p.row_bytes % 16 || p.src_rows <= 0 || p.mode < 0 ||
      p.mode > 1)
    return hipErrorInvalidValue;
  long long grid = (long long)device_cu_count() * 8;  // enough rows in flight for the full HBM rate
  if (max_wg > 0 && grid > max_wg) grid = max_wg;
  hipLaunchKernelGGL(ep_copy_kernel, dim3((unsigned)grid), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace moe
