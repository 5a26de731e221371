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
// experts are found by rounds of a wave-wide argmax on (key descending,
// index ascending), built from DPP lane exchanges within 16-lane rows and
// reads of the four row results.
#include "moe_internal.h"

namespace moe {
namespace {

// Tokens (one wave each) per workgroup, chosen per launch: one below
// kOneWaveTokens tokens, so a small batch spreads over as many compute units
// as it has tokens (128 tokens: 12.6 us in the layer against 18.0 with four
// per workgroup); four from there up, where single-wave workgroups made the
// kernel slower (4096 tokens: 27.2 us against 24-25).
constexpr int kOneWaveTokens = 1024;

struct KeyIdx {
  double key;
  int idx;
};

__device__ __forceinline__ bool better(double ka, int ia, double kb, int ib) {
  return ka > kb || (ka == kb && ia < ib);
}

// Wave-wide reductions. Four DPP steps combine the lanes of each 16-lane row
// (swap neighbours, swap pairs, mirror within 8 lanes, mirror within 16);
// the four row results are then read as wave-uniform values (lanes 0, 16,
// 32, 48) and combined in a fixed order, so every lane gets the same result.
// Every call is made with all 64 lanes active.
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;

template <int CTRL>
__device__ __forceinline__ int dpp_i32(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const uint64_t b = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = (uint32_t)dpp_i32<CTRL>((int)(uint32_t)b);
  const uint32_t hi = (uint32_t)dpp_i32<CTRL>((int)(uint32_t)(b >> 32));
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ double readlane_f64(double v, int lane) {
  const uint64_t b = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), lane);
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

template <int CTRL>
__device__ __forceinline__ void argmax_step(double& key, int& idx) {
  const double ok = dpp_f64<CTRL>(key);
  const int oi = dpp_i32<CTRL>(idx);
  if (better(ok, oi, key, idx)) {
    key = ok;
    idx = oi;
  }
}

__device__ __forceinline__ KeyIdx wave_argmax(double key, int idx) {
  argmax_step<kDppXor1>(key, idx);
  argmax_step<kDppXor2>(key, idx);
  argmax_step<kDppHalfMirror>(key, idx);
  argmax_step<kDppMirror>(key, idx);
  KeyIdx b{readlane_f64(key, 0), __builtin_amdgcn_readlane(idx, 0)};
#pragma unroll
  for (int r = 1; r < 4; ++r) {
    const double k = readlane_f64(key, 16 * r);
    const int i = __builtin_amdgcn_readlane(idx, 16 * r);
    if (better(k, i, b.key, b.idx)) {
      b.key = k;
      b.idx = i;
    }
  }
  return b;
}

__device__ __forceinline__ double wave_sum(double v) {
  v += dpp_f64<kDppXor1>(v);
  v += dpp_f64<kDppXor2>(v);
  v += dpp_f64<kDppHalfMirror>(v);
  v += dpp_f64<kDppMirror>(v);
  return (readlane_f64(v, 0) + readlane_f64(v, 16)) + (readlane_f64(v, 32) + readlane_f64(v, 48));
}

__device__ __forceinline__ double wave_max(double v) {
  v = fmax(v, dpp_f64<kDppXor1>(v));
  v = fmax(v, dpp_f64<kDppXor2>(v));
  v = fmax(v, dpp_f64<kDppHalfMirror>(v));
  v = fmax(v, dpp_f64<kDppMirror>(v));
  return fmax(fmax(readlane_f64(v, 0), readlane_f64(v, 16)), fmax(readlane_f64(v, 32), readlane_f64(v, 48)));
}

// Top two (as a multiset) of the keys held by a run of lanes: each lane
// starts with the top two of its own keys (m1 >= m2) and merges with a
// partner lane's pair at every step.
template <int CTRL>
__device__ __forceinline__ void top2_step(double& m1, double& m2) {
  const double b1 = dpp_f64<CTRL>(m1), b2 = dpp_f64<CTRL>(m2);
  const double n2 = (m1 >= b1) ? fmax(m2, b1) : fmax(m1, b2);
  m1 = fmax(m1, b1);
  m2 = n2;
}

template <int EPL, int kWaves>
__global__ void __launch_bounds__(64 * kWaves) route_kernel(RouteParams p) {
  __shared__ double skeys[kWaves][256];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int t = blockIdx.x * kWaves + wave;
  const bool active = t < p.T;  // inactive waves still reach every barrier
  const int E = p.E;
  const double NEG = -__builtin_inf();

  // ---- scores and keys ---------------------------------------------------
  double key[EPL], score[EPL];
  float u[EPL], bv[EPL];
  // Logits: the K-split partials summed in ascending split order. The first
  // split and the selection bias are loaded unconditionally, from indices
  // clamped into range, and dropped afterwards where they do not count (a
  // load under its own condition is waited for on its own). Each later round
  // issues the loads of up to 8 splits for all of the lane's experts before
  // adding them; those loads keep their conditions (clamped loads of the
  // splits past the last measured slower).
  {
    constexpr int R = 8;
    const size_t trow = (size_t)min(t, p.T - 1) * E;
    int ec[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) ec[i] = min(lane * EPL + i, E - 1);
    const float* const bias = p.bias ? p.bias : p.logits_in;  // any valid address when there is no bias
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      u[i] = p.logits_in[trow + ec[i]];
      bv[i] = bias[ec[i]];
    }
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const int e = lane * EPL + i;
      if (!(active && e < E)) u[i] = 0.f;
      if (!(p.bias && e < E)) bv[i] = 0.f;
    }
    for (int sp0 = 1; sp0 < p.nsplit; sp0 += R) {
      float part[R][EPL];
#pragma unroll
      for (int q = 0; q < R; ++q)
#pragma unroll
        for (int i = 0; i < EPL; ++i) {
          const int e = lane * EPL + i;
          part[q][i] = (active && e < E && sp0 + q < p.nsplit)
                           ? p.logits_in[(size_t)(sp0 + q) * p.split_stride + trow + e]
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
      key[i] = score[i] + (double)bv[i];
    } else {  // softmax: select on the logit; probabilities come later
      score[i] = (double)u[i];
      key[i] = (double)u[i];
    }
  }

  // ---- group limit ---------------------------------------------------------
  bool elig[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) elig[i] = (lane * EPL + i) < E;
  const int gs = p.n_groups > 1 ? E / p.n_groups : E;  // experts per group
  const int lpg = gs / EPL;                             // lanes per group when gs % EPL == 0
  if (p.n_groups > 1 && E == 64 * EPL && gs % EPL == 0 && (lpg == 2 || lpg == 4 || lpg == 8 || lpg == 16)) {
    // Every group is a run of lpg lanes. Its score (sum of its two largest
    // keys) comes from merging the lanes' top-two pairs within the run; the
    // groups are then ranked on the wave-uniform scores read from the first
    // lane of each run (score descending, index ascending), and a group is
    // kept when fewer than topk_groups groups rank above it.
    double m1 = NEG, m2 = NEG;
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const double v = key[i];
      if (v > m1) {
        m2 = m1;
        m1 = v;
      } else if (v > m2) {
        m2 = v;
      }
    }
    top2_step<kDppXor1>(m1, m2);
    if (lpg >= 4) top2_step<kDppXor2>(m1, m2);
    if (lpg >= 8) top2_step<kDppHalfMirror>(m1, m2);
    if (lpg >= 16) top2_step<kDppMirror>(m1, m2);
    const double gscore = m1 + m2;
    const int g = lane / lpg;
    int rank = 0;
    for (int h = 0; h < p.n_groups; ++h) {
      const double o = readlane_f64(gscore, h * lpg);
      if (better(o, h, gscore, g)) ++rank;
    }
    if (rank >= p.topk_groups) {
#pragma unroll
      for (int i = 0; i < EPL; ++i) elig[i] = false;
    }
  } else if (p.n_groups > 1) {
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if (lane * EPL + i < E) skeys[wave][lane * EPL + i] = key[i];
    __syncthreads();
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
    // the winner's score, read from the lane that holds it (w is wave-uniform)
    const int wl = (w.idx / EPL) & 63, wi = w.idx % EPL;
    double own = score[0];
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      if (i == wi) own = score[i];
      if (lane * EPL + i == w.idx) taken[i] = true;
    }
    const double sc = readlane_f64(own, wl);
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

template <int W>
void launch_epl(const RouteParams& p, int epl, hipStream_t s) {
  const dim3 grid((p.T + W - 1) / W), block(64 * W);
  switch (epl) {
    case 1: hipLaunchKernelGGL((route_kernel<1, W>), grid, block, 0, s, p); break;
    case 2: hipLaunchKernelGGL((route_kernel<2, W>), grid, block, 0, s, p); break;
    case 3: hipLaunchKernelGGL((route_kernel<3, W>), grid, block, 0, s, p); break;
    default: hipLaunchKernelGGL((route_kernel<4, W>), grid, block, 0, s, p); break;
  }
}

}  // namespace

hipError_t launch_route(const RouteParams& p, hipStream_t s) {
  if (p.T <= 0) return hipSuccess;
  const int epl = (p.E + 63) / 64;
  if (p.T < kOneWaveTokens) {
    launch_epl<1>(p, epl, s);
  } else {
    launch_epl<4>(p, epl, s);
  }
  return hipGetLastError();
}

}  // namespace moe
