// bf16 GEMMs with both operands k-contiguous: the input-gradient products
// dX = dY W^T and the attention scores Q K^T / dO V^T.
#include "gemm_bf16_kernel.h"

hipError_t gemm_bf16_nt(const GemmParams& p, hipStream_t s) {
  switch (p.epi) {
    case EPI_STORE: return launch_bf16<true, true, EPI_STORE>(p, s);
    case EPI_GELU_BWD: return launch_bf16<true, true, EPI_GELU_BWD>(p, s);
    case EPI_F32_STORE: return launch_bf16<true, true, EPI_F32_STORE>(p, s);
    default: return hipErrorInvalidValue;
  }
}
