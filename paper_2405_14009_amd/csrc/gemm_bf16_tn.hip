// bf16 GEMMs with both operands m/n-contiguous: the weight-gradient products
// dW = X^T dY (reduction over tokens, fp32 accumulate into the gradient
// buffers) and the attention products P^T dO, dS^T Q.
#include "gemm_bf16_kernel.h"

namespace {

// out[n] (+)= sum over the rows r of work[r][n], in row order.  Rows are
// requested 16 at a time and then added in order (one load in flight per
// thread made the 64-row sums of a 16384-row product take 30 us).
__global__ __launch_bounds__(256) void colsum_rows_k(const float* __restrict__ work, int rows, int n,
                                                     float* __restrict__ out, int accumulate) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= n) return;
  float t = 0.f;
  int r = 0;
  for (; r + 16 <= rows; r += 16) {
    float v[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = work[(long)(r + i) * n + c];
#pragma unroll
    for (int i = 0; i < 16; ++i) t += v[i];
  }
  for (; r < rows; ++r) t += work[(long)r * n + c];
  out[c] = (accumulate ? out[c] : 0.f) + t;
}

}  // namespace

hipError_t gemm_bf16_tn(const GemmParams& p, hipStream_t s) {
  hipError_t e;
  switch (p.epi) {
    case EPI_STORE: e = launch_bf16<false, false, EPI_STORE>(p, s); break;
    case EPI_F32_ACC: e = launch_bf16<false, false, EPI_F32_ACC>(p, s); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess || p.colsum_out == nullptr) return e;
  hipLaunchKernelGGL(colsum_rows_k, dim3((p.N + 255) / 256), dim3(256), 0, s, p.colsum_work,
                     (p.M + 255) / 256, p.N, p.colsum_out, p.colsum_acc);
  return hipGetLastError();
}
