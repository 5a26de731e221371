// Top-k routing: one wavefront per token.
//
// The paper's MoE workload routes every token to its experts before the
// dispatch (App. M); the rule implemented is the public DeepSeek-V3 one
// (sigmoid scores, per-expert selection bias, group-limited top-k, weights
// from the unbiased scores, normalised and scaled) or the Mixtral one
// (softmax, top-k, renormalised).
//
// Lane l holds experts [l*EPL, l*EPL + EPL) (EPL = ceil(E/64) <= 4), so the
// logits of a token are read with one coalesced load per lane. When the
// router GEMM was split along K, the kernel first sums the partial logits in
// a fixed order (and stores the sums), so the logits stay deterministic. Keys, group
// scores and weights are evaluated in fp64: the selection is then a
// deterministic function of the fp32 logits' bits and a near-tie in fp32
// cannot flip it. Group scores (sum of a group's two largest keys) come from
// a per-wave LDS copy of the keys; the best groups and then the k best
// experts are found by k rounds of a wave-wide butterfly argmax on
// (key descending, index ascending).
#include "moe_internal.h"

namespace moe {
namespace {

constexpr int kWaves = 4;

struct KeyIdx {
  double key;
  int idx;
};

__device__ __forceinline__ bool better(double ka, int ia, double kb, int ib) {
  return ka > kb || (ka == kb && ia < ib);
}

__device__ __forceinline__ KeyIdx wave_argmax(double key, int idx) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const double ok = __shfl_xor(key, o, 64);
    const int oi = __shfl_xor(idx, o, 64);
    if (better(ok, oi, key, idx)) {
      key = ok;
      idx = oi;
    }
  }
  return {key, idx};
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ double wave_max(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmax(v, __shfl_xor(v, o, 64));
  return v;
}

template <int EPL>
__global__ void __launch_bounds__(64 * kWaves) route_kernel(RouteParams p) {
  __shared__ double skeys[kWaves][256];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int t = blockIdx.x * kWaves + wave;
  const bool active = t < p.T;  // inactive waves still reach every barrier
  const int E = p.E;
  const double NEG = -__builtin_inf();

  // ---- scores and keys ---------------------------------------------------
  double key[EPL], score[EPL];
  float u[EPL];
  // Logits: the K-split partials summed in ascending split order. Each
  // round issues the loads of up to 8 splits for all of the lane's experts
  // before adding them, so the loads overlap instead of waiting one by one.
  {
    constexpr int R = 8;
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const int e = lane * EPL + i;
      u[i] = (active && e < E) ? p.logits_in[(size_t)t * E + e] : 0.f;
    }
    for (int sp0 = 1; sp0 < p.nsplit; sp0 += R) {
      float part[R][EPL];
#pragma unroll
      for (int q = 0; q < R; ++q)
#pragma unroll
        for (int i = 0; i < EPL; ++i) {
          const int e = lane * EPL + i;
          part[q][i] = (active && e < E && sp0 + q < p.nsplit)
                           ? p.logits_in[(size_t)(sp0 + q) * p.split_stride + (size_t)t * E + e]
                           : 0.f;
        }
#pragma unroll
      for (int q = 0; q < R; ++q)
#pragma unroll
        for (int i = 0; i < EPL; ++i)
          if (sp0 + q < p.nsplit) u[i] += part[q][i];
    }
  }
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int e = lane * EPL + i;
    const bool ok = active && e < E;
    if (ok && p.logits_out) p.logits_out[(size_t)t * E + e] = u[i];
    if (!ok) {
      key[i] = NEG;
      score[i] = 0.0;
    } else if (p.score == 1) {  // sigmoid
      score[i] = 1.0 / (1.0 + exp(-(double)u[i]));
      key[i] = score[i] + (p.bias ? (double)p.bias[e] : 0.0);
    } else {  // softmax: select on the logit; probabilities come later
      score[i] = (double)u[i];
      key[i] = (double)u[i];
    }
  }

  // ---- group limit ---------------------------------------------------------
  bool elig[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) elig[i] = (lane * EPL + i) < E;
  if (p.n_groups > 1) {
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if (lane * EPL + i < E) skeys[wave][lane * EPL + i] = key[i];
    __syncthreads();
    const int gs = E / p.n_groups;
    double gscore = NEG;
    if (lane < p.n_groups) {
      double m1 = NEG, m2 = NEG;
      for (int e = lane * gs; e < (lane + 1) * gs; ++e) {
        const double v = skeys[wave][e];
        if (v > m1) {
          m2 = m1;
          m1 = v;
        } else if (v > m2) {
          m2 = v;
        }
      }
      gscore = (gs == 1) ? m1 : m1 + m2;
    }
    bool chosen = false;
    for (int r = 0; r < p.topk_groups; ++r) {
      const double c = (lane < p.n_groups && !chosen) ? gscore : NEG;
      const KeyIdx w = wave_argmax(c, lane < p.n_groups ? lane : 1 << 20);
      if (lane == w.idx) chosen = true;
    }
    const unsigned long long gmask = __ballot(chosen);
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const int e = lane * EPL + i;
      if (e < E && !((gmask >> (e / gs)) & 1ull)) elig[i] = false;
    }
  }

  // ---- top-k -----------------------------------------------------------------
  bool taken[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) taken[i] = false;
  int my_e = -1;         // lane j < k keeps slot j
  double my_score = 0.0;
  for (int j = 0; j < p.k; ++j) {
    double bk = NEG;
    int bi = 1 << 20;
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const int e = lane * EPL + i;
      if (elig[i] && !taken[i] && better(key[i], e, bk, bi)) {
        bk = key[i];
        bi = e;
      }
    }
    const KeyIdx w = wave_argmax(bk, bi);
    double sc = 0.0;
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if (lane * EPL + i == w.idx) {
        taken[i] = true;
        sc = score[i];
      }
    sc = wave_sum(sc);  // exactly one lane holds the winner's score
    if (lane == j) {
      my_e = w.idx;
      my_score = sc;
    }
  }

  // ---- weights ---------------------------------------------------------------
  double wgt = 0.0;
  const bool slot = lane < p.k;
  if (p.score == 1) {
    wgt = slot ? my_score : 0.0;
    if (p.renorm) wgt = wgt / wave_sum(wgt);
  } else {
    if (p.renorm) {
      const double m = __shfl(my_score, 0, 64);  // slot 0 holds the largest selected logit
      const double z = slot ? exp(my_score - m) : 0.0;
      wgt = z / wave_sum(z);
    } else {
      double mx = NEG;
#pragma unroll
      for (int i = 0; i < EPL; ++i)
        if (lane * EPL + i < E) mx = fmax(mx, (double)u[i]);
      mx = wave_max(mx);
      double zs = 0.0;
#pragma unroll
      for (int i = 0; i < EPL; ++i)
        if (lane * EPL + i < E) zs += exp((double)u[i] - mx);
      zs = wave_sum(zs);
      wgt = slot ? exp(my_score - mx) / zs : 0.0;
    }
  }
  wgt *= (double)p.scale;
  if (active && slot) {
    p.topk_idx[(size_t)t * p.k + lane] = my_e;
    p.topk_w[(size_t)t * p.k + lane] = (float)wgt;
  }
}

}  // namespace

hipError_t launch_route(const RouteParams& p, hipStream_t s) {
  if (p.T <= 0) return hipSuccess;
  const dim3 grid((p.T + kWaves - 1) / kWaves), block(64 * kWaves);
  const int epl = (p.E + 63) / 64;
  switch (epl) {
    case 1: hipLaunchKernelGGL(route_kernel<1>, grid, block, 0, s, p); break;
    case 2: hipLaunchKernelGGL(route_kernel<2>, grid, block, 0, s, p); break;
    case 3: hipLaunchKernelGGL(route_kernel<3>, grid, block, 0, s, p); break;
    default: hipLaunchKernelGGL(route_kernel<4>, grid, block, 0, s, p); break;
  }
  return hipGetLastError();
}

}  // namespace moe
