// Row softmax of the attention scores and its backward, over materialised
// score rows (one workgroup per (sequence, head, query) row, fp32 statistics,
// wavefront-shuffle reductions).  Entries after the query are masked to
// probability 0 when causal; masked and padded entries are written as 0 so
// the following products can read whole tiles.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace {

constexpr int NT = 256;

template <class E>
__global__ __launch_bounds__(NT) void softmax_fwd_k(const float* __restrict__ S, E* __restrict__ P,
                                                    int s, float scale, int causal) {
  __shared__ float red[NT / 64];
  const long r = blockIdx.x;
  const int q = (int)(r % s);
  const int len = causal ? q + 1 : s;
  const float* sr = S + r * s;
  E* pr = P + r * s;
  float mx = -INFINITY;
  for (int c = threadIdx.x; c < len; c += NT) mx = fmaxf(mx, sr[c] * scale);
  mx = block_max<NT>(mx, red);
  float sum = 0.f;
  for (int c = threadIdx.x; c < len; c += NT) sum += expf(sr[c] * scale - mx);
  sum = block_sum<NT>(sum, red);
  const float inv = 1.0f / sum;
  for (int c = threadIdx.x; c < s; c += NT)
    pr[c] = from_f32<E>(c < len ? expf(sr[c] * scale - mx) * inv : 0.f);
}

template <class E>
__global__ __launch_bounds__(NT) void softmax_bwd_k(const float* __restrict__ dP,
                                                    const E* __restrict__ P, E* __restrict__ dS,
                                                    int s, float scale, int causal) {
  __shared__ float red[NT / 64];
  const long r = blockIdx.x;
  const int q = (int)(r % s);
  const int len = causal ? q + 1 : s;
  const float* dpr = dP + r * s;
  const E* pr = P + r * s;
  E* out = dS + r * s;
  float d = 0.f;
  for (int c = threadIdx.x; c < len; c += NT) d += dpr[c] * to_f32(pr[c]);
  d = block_sum<NT>(d, red);
  for (int c = threadIdx.x; c < s; c += NT)
    out[c] = from_f32<E>(c < len ? scale * to_f32(pr[c]) * (dpr[c] - d) : 0.f);
}

}  // namespace

hipError_t softmax_forward(int elt, const float* S, void* P, long rows, int s, float scale,
                           int causal, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  if (elt == 2)
    hipLaunchKernelGGL(softmax_fwd_k<bf16>, dim3(rows), dim3(NT), 0, st, S, (bf16*)P, s, scale, causal);
  else
    hipLaunchKernelGGL(softmax_fwd_k<float>, dim3(rows), dim3(NT), 0, st, S, (float*)P, s, scale, causal);
  return hipGetLastError();
}

hipError_t softmax_backward(int elt, const float* dP, const void* P, void* dS, long rows, int s,
                            float scale, int causal, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  if (elt == 2)
    hipLaunchKernelGGL(softmax_bwd_k<bf16>, dim3(rows), dim3(NT), 0, st, dP, (const bf16*)P,
                       (bf16*)dS, s, scale, causal);
  else
    hipLaunchKernelGGL(softmax_bwd_k<float>, dim3(rows), dim3(NT), 0, st, dP, (const float*)P,
                       (float*)dS, s, scale, causal);
  return hipGetLastError();
}
