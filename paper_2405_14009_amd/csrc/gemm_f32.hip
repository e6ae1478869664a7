// fp32 GEMM (vector ALU, fp32 FMA) for stages stored in fp32.  Same operand
// conventions, batching, causal k-ranges and epilogues as the bf16 MFMA
// family; 64x64 output tile, k-step 16, 4x4 outputs per thread.
#include "gemm.h"

namespace {

constexpr int TB = 64, TK = 16, NT = 256;

template <bool AK, bool BKC, int EPI>
__global__ __launch_bounds__(NT) void gemm_f32_kernel(GemmParams p) {
  __shared__ float sA[TK][TB + 4];
  __shared__ float sB[TK][TB + 4];
  const int tiles_m = (p.M + TB - 1) / TB;
  const int tm = blockIdx.x % tiles_m, tn = blockIdx.x / tiles_m;
  const int m0 = tm * TB, n0 = tn * TB;
  if (p.causal_skip && n0 > m0 + TB - 1) return;
  const int z = blockIdx.y, zb = z / p.heads, zh = z % p.heads;
  const float* A = (const float*)p.A + zb * p.a_bs + zh * p.a_hs;
  const float* B = (const float*)p.B + zb * p.b_bs + zh * p.b_hs;
  const long c_off = zb * p.c_bs + zh * p.c_hs;
  int kb = 0, ke = p.K;
  if (p.krange == KR_BELOW) ke = min(p.K, m0 + TB);
  else if (p.krange == KR_ABOVE) kb = (m0 / TK) * TK;

  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  float acc[4][4] = {};
  for (int k0 = kb; k0 < ke; k0 += TK) {
#pragma unroll
    for (int i = 0; i < (TB * TK) / NT; ++i) {
      const int e = tid + i * NT;
      int mm, kk;
      if (AK) { mm = e / TK; kk = e % TK; } else { kk = e / TB; mm = e % TB; }
      const int m = m0 + mm, k = k0 + kk;
      float va = 0.f;
      if (m < p.M && k < ke) {
        const float* a = A;
        int kl = k;
        if (p.kseg_len > 0) {
          a = (const float*)p.segA[k / p.kseg_len] + zb * p.a_bs + zh * p.a_hs;
          kl = k % p.kseg_len;
        }
        va = AK ? a[(long)m * p.lda + kl] : a[(long)kl * p.lda + m];
      }
      sA[kk][mm] = va;
      int nn;
      if (BKC) { nn = e / TK; kk = e % TK; } else { kk = e / TB; nn = e % TB; }
      const int n = n0 + nn, k2 = k0 + kk;
      float vb = 0.f;
      if (n < p.N && k2 < ke) {
        const float* b = B;
        int kl = k2;
        if (p.kseg_len > 0) {
          b = (const float*)p.segB[k2 / p.kseg_len] + zb * p.b_bs + zh * p.b_hs;
          kl = k2 % p.kseg_len;
        }
        vb = BKC ? b[(long)n * p.ldb + kl] : b[(long)kl * p.ldb + n];
      }
      sB[kk][nn] = vb;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < TK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = sA[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = sB[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
  float* C = (float*)p.C + c_off;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + ty * 4 + i, n = n0 + tx * 4 + j;
      if (m < p.M && n < p.N) epi_store<EPI, float>(p, C, m, n, acc[i][j]);
    }
}

template <bool AK, bool BKC>
hipError_t launch_epi(const GemmParams& p, hipStream_t s) {
  dim3 grid(((p.M + TB - 1) / TB) * ((p.N + TB - 1) / TB), p.batch * p.heads);
  switch (p.epi) {
    case EPI_STORE: hipLaunchKernelGGL((gemm_f32_kernel<AK, BKC, EPI_STORE>), grid, dim3(NT), 0, s, p); break;
    case EPI_BIAS: hipLaunchKernelGGL((gemm_f32_kernel<AK, BKC, EPI_BIAS>), grid, dim3(NT), 0, s, p); break;
    case EPI_BIAS_RESID: hipLaunchKernelGGL((gemm_f32_kernel<AK, BKC, EPI_BIAS_RESID>), grid, dim3(NT), 0, s, p); break;
    case EPI_BIAS_GELU: hipLaunchKernelGGL((gemm_f32_kernel<AK, BKC, EPI_BIAS_GELU>), grid, dim3(NT), 0, s, p); break;
    case EPI_GELU_BWD: hipLaunchKernelGGL((gemm_f32_kernel<AK, BKC, EPI_GELU_BWD>), grid, dim3(NT), 0, s, p); break;
    case EPI_F32_ACC: hipLaunchKernelGGL((gemm_f32_kernel<AK, BKC, EPI_F32_ACC>), grid, dim3(NT), 0, s, p); break;
    default: hipLaunchKernelGGL((gemm_f32_kernel<AK, BKC, EPI_F32_STORE>), grid, dim3(NT), 0, s, p); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t gemm_f32(const GemmParams& p, hipStream_t s) {
  if (p.M <= 0 || p.N <= 0 || p.batch * p.heads <= 0) return hipSuccess;
  if (p.kseg_len > 0 && (p.K % p.kseg_len || p.K / p.kseg_len > GEMM_MAX_SEG)) return hipErrorInvalidValue;
  if (p.colsum_out != nullptr) return hipErrorInvalidValue;  // bf16 products only
  if (p.a_kcontig && !p.b_kcontig) return launch_epi<true, false>(p, s);
  if (p.a_kcontig && p.b_kcontig) return launch_epi<true, true>(p, s);
  if (!p.a_kcontig && !p.b_kcontig) return launch_epi<false, false>(p, s);
  return launch_epi<false, true>(p, s);
}
