// bf16 GEMMs with both operands m/n-contiguous: the weight-gradient products
// dW = X^T dY (reduction over tokens, fp32 accumulate into the gradient
// buffers) and the attention products P^T dO, dS^T Q.
#include "gemm_bf16_kernel.h"

hipError_t gemm_bf16_tn(const GemmParams& p, hipStream_t s) {
  switch (p.epi) {
    case EPI_STORE: return launch_bf16<false, false, EPI_STORE>(p, s);
    case EPI_F32_ACC: return launch_bf16<false, false, EPI_F32_ACC>(p, s);
    default: return hipErrorInvalidValue;
  }
}
