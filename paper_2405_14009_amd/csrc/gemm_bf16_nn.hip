// bf16 GEMMs with A k-contiguous and B n-contiguous (forward Y = X W, and
// the attention products P V and dS K), plus the top-level bf16 dispatcher.
#include "gemm_bf16_kernel.h"

hipError_t gemm_bf16_nt(const GemmParams& p, hipStream_t s);
hipError_t gemm_bf16_tn(const GemmParams& p, hipStream_t s);

static hipError_t gemm_bf16_nn(const GemmParams& p, hipStream_t s) {
  switch (p.epi) {
    case EPI_STORE: return launch_bf16<true, false, EPI_STORE>(p, s);
    case EPI_BIAS: return launch_bf16<true, false, EPI_BIAS>(p, s);
    case EPI_BIAS_RESID: return launch_bf16<true, false, EPI_BIAS_RESID>(p, s);
    case EPI_BIAS_GELU: return launch_bf16<true, false, EPI_BIAS_GELU>(p, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t gemm_bf16(const GemmParams& p, hipStream_t s) {
  if (p.M <= 0 || p.N <= 0 || p.batch * p.heads <= 0) return hipSuccess;
  // a segmented reduction needs whole 64-deep k-tiles per segment
  if (p.kseg_len > 0 && (p.kseg_len % 64 || p.K % p.kseg_len || p.K / p.kseg_len > GEMM_MAX_SEG ||
                         p.krange != KR_FULL))
    return hipErrorInvalidValue;
  if (p.a_kcontig && !p.b_kcontig) return gemm_bf16_nn(p, s);
  // column sums of B: weight-gradient layout only, with its workspace
  if (p.colsum_out != nullptr && (p.a_kcontig || p.b_kcontig || p.colsum_work == nullptr || p.batch * p.heads != 1))
    return hipErrorInvalidValue;
  if (p.a_kcontig && p.b_kcontig) return gemm_bf16_nt(p, s);
  if (!p.a_kcontig && !p.b_kcontig) return gemm_bf16_tn(p, s);
  return hipErrorInvalidValue;
}
