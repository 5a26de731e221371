// fp32 grouped GEMM on the vector ALU, for the fp32 configurations.
//
// Same problem as the bf16 matrix-core kernel (the expert FFN of App. M step
// 3 and the router GEMM): row r of the output reads A row gather[r] and uses
// the weights of the group that owns r. Each 16x16 output tile is computed by
// one workgroup from 16x32 operand slices staged in LDS; every output element
// accumulates its dot product in fp32 in ascending k. This path serves small
// fp32 problems, where the matrix cores bring nothing.
#include "moe_internal.h"

namespace moe {
namespace {

constexpr int TS = 16;  // output tile edge
constexpr int KS = 32;  // k slice

__device__ __forceinline__ int group_of_row(const int32_t* offsets, int groups, int row) {
  int lo = 0, hi = groups - 1;  // largest g with offsets[g] <= row
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (offsets[mid] <= row) lo = mid; else hi = mid - 1;
  }
  return lo;
}

template <int EPI>
__global__ void __launch_bounds__(TS * TS) gemm_f32_kernel(GemmProblem p) {
  __shared__ float as[TS][KS + 1];
  const int tx = threadIdx.x % TS, ty = threadIdx.x / TS;
  const int row_base = blockIdx.y * TS;
  const int col_base = blockIdx.x * TS;
  const int M = p.offsets ? min(max(p.offsets[p.groups], 0), p.M) : p.M;
  if (row_base >= M) return;

  // Rows of one tile may belong to different groups, so B is fetched per
  // output row: the thread (ty, tx) computes C[row_base+ty][col_base+tx] and
  // the tile loads B rows for its columns once per distinct group.
  const int row = row_base + ty;
  const bool row_ok = row < M;
  const int g = (p.offsets && row_ok) ? group_of_row(p.offsets, p.groups, row) : 0;
  const float* A = static_cast<const float*>(p.A);
  const size_t K = (size_t)p.K;
  const int arow = row_ok ? (p.gather ? min(max(p.gather[row], 0), p.a_rows - 1) : row) : 0;
  const int col = col_base + tx;
  const size_t gstride = (size_t)p.N * K;
  const float* B0 = static_cast<const float*>(p.B0) + (size_t)g * gstride;
  const float* B1 = (EPI == EPI_SWIGLU) ? static_cast<const float*>(p.B1) + (size_t)g * gstride : nullptr;

  float acc0 = 0.f, acc1 = 0.f;
  for (int k0 = 0; k0 < p.K; k0 += KS) {
    // stage this thread's A row slice (each row's 32 values loaded by 16 threads)
    for (int kk = tx; kk < KS; kk += TS) as[ty][kk] = (row_ok && k0 + kk < p.K) ? A[(size_t)arow * K + k0 + kk] : 0.f;
    __syncthreads();
    if (row_ok && col < p.N) {
      const float* b0 = B0 + (size_t)col * K + k0;
      const float* b1 = (EPI == EPI_SWIGLU) ? B1 + (size_t)col * K + k0 : nullptr;
      const int kend = min(KS, p.K - k0);
      for (int kk = 0; kk < kend; ++kk) {
        acc0 = fmaf(as[ty][kk], b0[kk], acc0);
        if (EPI == EPI_SWIGLU) acc1 = fmaf(as[ty][kk], b1[kk], acc1);
      }
    }
    __syncthreads();
  }
  if (!row_ok || col >= p.N) return;
  float* C = static_cast<float*>(p.C);
  float v = acc0;
  if (EPI == EPI_SWIGLU) v = acc0 / (1.0f + expf(-acc0)) * acc1;
  C[(size_t)row * p.ldc + col] = v;
}

}  // namespace

hipError_t launch_gemm_f32(const GemmProblem& p, int epi, hipStream_t s) {
  if (p.M <= 0 || p.N <= 0) return hipSuccess;
  dim3 grid((p.N + TS - 1) / TS, (p.M + TS - 1) / TS);
  if (epi == EPI_SWIGLU)
    hipLaunchKernelGGL(gemm_f32_kernel<EPI_SWIGLU>, grid, dim3(TS * TS), 0, s, p);
  else
    hipLaunchKernelGGL(gemm_f32_kernel<EPI_STORE>, grid, dim3(TS * TS), 0, s, p);
  return hipGetLastError();
}

}  // namespace moe
