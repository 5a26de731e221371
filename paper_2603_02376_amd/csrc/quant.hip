// Per-token quantization of the token rows (the pipeline of App. F
// quantizes the tokens to int8 with one scale per token before the dispatch
// exchange and dequantizes them on the expert side before GEMM1; Table 5
// names an FP8 quantize phase).
//
// int8:  scale[t] = max_c |x[t, c]| / 127          (fp32, IEEE division)
//        codes[t, c] = rne(x[t, c] / scale[t])     (fp32 division, round half
//                                                   to even, clamped to +-127)
// FP8 (OCP E4M3: bias 7, largest value 448, 0x7F NaN):
//        scale[t] = max_c |x[t, c]| / 448
//        codes[t, c] = E4M3 of x[t, c] / scale[t]  (fp32 quotient clamped to
//                                                   +-448, then the hardware
//                                                   conversion, round to
//                                                   nearest even; it does not
//                                                   saturate, hence the clamp)
// A row of zeros gets scale 0 and codes 0. One wave per token row: each lane
// reads 8 bf16 (16 bytes) at a time (rows of up to 8192 elements are loaded
// whole into registers first), the wave reduces the row's maximum with
// butterfly shuffles, then every lane writes its 8 codes as one 8-byte store.
#include "moe_internal.h"

namespace moe {
namespace {

constexpr int kWavesQ = 4;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// 8 codes of 8 consecutive elements (one 16-byte chunk of bf16) at scale > 0.
template <bool FP8>
__device__ __forceinline__ uint2 quantize8(uint4 v, float scale) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  uint32_t out[2] = {0u, 0u};
  if constexpr (FP8) {
    // element 2i in the low bf16 of w[i], 2i+1 in the high one; the
    // conversion puts its first operand in the lower byte of the half
    // word it writes (word_sel false: bytes 0-1, true: bytes 2-3)
    float a[4], b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      a[i] = fminf(fmaxf(bf16_lo(w[i]) / scale, -448.f), 448.f);
      b[i] = fminf(fmaxf(bf16_hi(w[i]) / scale, -448.f), 448.f);
    }
    out[0] = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a[0], b[0], 0, false);
    out[0] = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a[1], b[1], (int)out[0], true);
    out[1] = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a[2], b[2], 0, false);
    out[1] = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a[3], b[3], (int)out[1], true);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float f[2] = {bf16_lo(w[i]), bf16_hi(w[i])};
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float q = fminf(fmaxf(rintf(f[h] / scale), -127.f), 127.f);
        const uint32_t b = (uint32_t)((int)q) & 0xFFu;
        out[i / 2] |= b << (8 * (2 * (i % 2) + h));
      }
    }
  }
  return make_uint2(out[0], out[1]);
}

__device__ __forceinline__ float absmax8(uint4 v, float m) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) m = fmaxf(m, fmaxf(fabsf(bf16_lo(w[i])), fabsf(bf16_hi(w[i]))));
  return m;
}

// CPL > 0: the row (at most 64 * CPL chunks) is held in registers, CPL
// chunks per lane, all loaded before the maximum is taken; CPL == 0: any
// width, the row is read twice.
template <bool FP8, int CPL>
__global__ void __launch_bounds__(64 * kWavesQ) quantize_kernel(const __bf16* __restrict__ x, int8_t* __restrict__ codes,
                                                               float* __restrict__ scales, int T, int d) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * kWavesQ + (threadIdx.x >> 6);
  if (row >= T) return;
  const uint4* src = reinterpret_cast<const uint4*>(x + (size_t)row * d);
  const int n8 = d / 8;  // 16-byte chunks per row (d % 64 == 0)
  uint2* dst = reinterpret_cast<uint2*>(codes + (size_t)row * d);
  float m = 0.f;
  uint4 v[CPL > 0 ? CPL : 1];
  if constexpr (CPL > 0) {
#pragma unroll
    for (int i = 0; i < CPL; ++i) v[i] = (lane + 64 * i < n8) ? src[lane + 64 * i] : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
    for (int i = 0; i < CPL; ++i) m = absmax8(v[i], m);
  } else {
    for (int c = lane; c < n8; c += 64) m = absmax8(src[c], m);
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
  const float scale = m / (FP8 ? 448.0f : 127.0f);
  if (lane == 0) scales[row] = scale;
  if constexpr (CPL > 0) {
#pragma unroll
    for (int i = 0; i < CPL; ++i)
      if (lane + 64 * i < n8) dst[lane + 64 * i] = scale > 0.f ? quantize8<FP8>(v[i], scale) : make_uint2(0u, 0u);
  } else {
    for (int c = lane; c < n8; c += 64) dst[c] = scale > 0.f ? quantize8<FP8>(src[c], scale) : make_uint2(0u, 0u);
  }
}

}  // namespace

hipError_t launch_quantize(const void* x, int8_t* codes, float* scales, int T, int d, bool fp8, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  if (d <= 0 || d % 64 != 0) return hipErrorInvalidValue;
  const unsigned grid = (unsigned)((T + kWavesQ - 1) / kWavesQ);
  constexpr int kCpl = 16;  // rows of up to 8192 elements stay in registers
  auto kern = d <= 512 * kCpl ? (fp8 ? quantize_kernel<true, kCpl> : quantize_kernel<false, kCpl>)
                              : (fp8 ? quantize_kernel<true, 0> : quantize_kernel<false, 0>);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(64 * kWavesQ), 0, s, static_cast<const __bf16*>(x), codes, scales, T, d);
  return hipGetLastError();
}

}  // namespace moe
