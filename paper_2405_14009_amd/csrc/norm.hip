// LayerNorm forward / input-gradient kernels (one workgroup per token row,
// fp32 statistics, wavefront-shuffle reductions) and the deterministic
// column reductions of the weight pass (bias and LayerNorm-affine gradients).
#include "common.h"
#include "kernels.h"

namespace {

constexpr int NT = 256;
constexpr int CHUNK = 64;  // rows per partial sum of the column reductions

template <class E>
__global__ __launch_bounds__(NT) void ln_fwd_k(const E* __restrict__ x, const float* __restrict__ g,
                                               const float* __restrict__ b, E* __restrict__ y,
                                               float* __restrict__ mean, float* __restrict__ rstd,
                                               int h, float eps) {
  __shared__ float red[NT / 64];
  const long row = blockIdx.x;
  const E* xr = x + row * h;
  E* yr = y + row * h;
  float s = 0.f;
  for (int c = threadIdx.x; c < h; c += NT) s += to_f32(xr[c]);
  const float mu = block_sum<NT>(s, red) / h;
  float q = 0.f;
  for (int c = threadIdx.x; c < h; c += NT) {
    const float d = to_f32(xr[c]) - mu;
    q += d * d;
  }
  const float var = block_sum<NT>(q, red) / h;
  const float rs = 1.0f / sqrtf(var + eps);
  for (int c = threadIdx.x; c < h; c += NT) yr[c] = from_f32<E>((to_f32(xr[c]) - mu) * rs * g[c] + b[c]);
  if (threadIdx.x == 0) {
    mean[row] = mu;
    rstd[row] = rs;
  }
}

template <class E>
__global__ __launch_bounds__(NT) void ln_bwd_k(const E* __restrict__ dout, const E* __restrict__ x,
                                               const float* __restrict__ mean,
                                               const float* __restrict__ rstd,
                                               const float* __restrict__ g,
                                               const E* __restrict__ resid, E* __restrict__ dx, int h) {
  __shared__ float red[NT / 64];
  const long row = blockIdx.x;
  const float mu = mean[row], rs = rstd[row];
  const E* dr = dout + row * h;
  const E* xr = x + row * h;
  float s1 = 0.f, s2 = 0.f;
  for (int c = threadIdx.x; c < h; c += NT) {
    const float xh = (to_f32(xr[c]) - mu) * rs;
    const float dz = to_f32(dr[c]) * g[c];
    s1 += dz;
    s2 += dz * xh;
  }
  const float m1 = block_sum<NT>(s1, red) / h;
  const float m2 = block_sum<NT>(s2, red) / h;
  const E* rr = resid + row * h;
  E* out = dx + row * h;
  for (int c = threadIdx.x; c < h; c += NT) {
    const float xh = (to_f32(xr[c]) - mu) * rs;
    const float dz = to_f32(dr[c]) * g[c];
    out[c] = from_f32<E>(to_f32(rr[c]) + rs * (dz - m1 - xh * m2));
  }
}

template <class E, bool LN>
__global__ __launch_bounds__(NT) void colsum_part_k(const E* __restrict__ dout, long ld,
                                                    const E* __restrict__ x,
                                                    const float* __restrict__ mean,
                                                    const float* __restrict__ rstd, long rows,
                                                    int n, float* __restrict__ part_b,
                                                    float* __restrict__ part_g) {
  const int c = blockIdx.x * NT + threadIdx.x;
  if (c >= n) return;
  const long r0 = (long)blockIdx.y * CHUNK;
  const long r1 = min(rows, r0 + CHUNK);
  float sb = 0.f, sg = 0.f;
  for (long r = r0; r < r1; ++r) {
    const float d = to_f32(dout[r * ld + c]);
    sb += d;
    if (LN) sg += d * (to_f32(x[r * n + c]) - mean[r]) * rstd[r];
  }
  part_b[(long)blockIdx.y * n + c] = sb;
  if (LN) part_g[(long)blockIdx.y * n + c] = sg;
}

__global__ __launch_bounds__(NT) void colsum_final_k(const float* __restrict__ part, int nchunk,
                                                     int n, float* __restrict__ out, int accumulate) {
  const int c = blockIdx.x * NT + threadIdx.x;
  if (c >= n) return;
  float s = 0.f;
  for (int ch = 0; ch < nchunk; ++ch) s += part[(long)ch * n + c];
  out[c] = accumulate ? out[c] + s : s;
}

}  // namespace

hipError_t ln_forward(int elt, const void* x, const float* g, const float* b, void* y, float* mean,
                      float* rstd, long rows, int h, float eps, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (elt == 2)
    hipLaunchKernelGGL(ln_fwd_k<bf16>, dim3(rows), dim3(NT), 0, s, (const bf16*)x, g, b, (bf16*)y,
                       mean, rstd, h, eps);
  else
    hipLaunchKernelGGL(ln_fwd_k<float>, dim3(rows), dim3(NT), 0, s, (const float*)x, g, b,
                       (float*)y, mean, rstd, h, eps);
  return hipGetLastError();
}

hipError_t ln_backward(int elt, const void* dout, const void* x, const float* mean,
                       const float* rstd, const float* g, const void* resid, void* dx, long rows,
                       int h, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (elt == 2)
    hipLaunchKernelGGL(ln_bwd_k<bf16>, dim3(rows), dim3(NT), 0, s, (const bf16*)dout, (const bf16*)x,
                       mean, rstd, g, (const bf16*)resid, (bf16*)dx, h);
  else
    hipLaunchKernelGGL(ln_bwd_k<float>, dim3(rows), dim3(NT), 0, s, (const float*)dout,
                       (const float*)x, mean, rstd, g, (const float*)resid, (float*)dx, h);
  return hipGetLastError();
}

long colsum_part_floats(long rows, int n) { return 2 * ((rows + CHUNK - 1) / CHUNK) * (long)n; }

static hipError_t colsum_impl(int elt, bool ln, const void* dout, long ld, const void* x,
                              const float* mean, const float* rstd, long rows, int n, float* dg,
                              float* db, int accumulate, float* part, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int nchunk = (int)((rows + CHUNK - 1) / CHUNK);
  float* part_b = part;
  float* part_g = part + (long)nchunk * n;
  dim3 grid((n + NT - 1) / NT, nchunk);
  if (nchunk > 0) {
    if (elt == 2) {
      if (ln)
        hipLaunchKernelGGL((colsum_part_k<bf16, true>), grid, dim3(NT), 0, s, (const bf16*)dout, ld,
                           (const bf16*)x, mean, rstd, rows, n, part_b, part_g);
      else
        hipLaunchKernelGGL((colsum_part_k<bf16, false>), grid, dim3(NT), 0, s, (const bf16*)dout, ld,
                           (const bf16*)nullptr, mean, rstd, rows, n, part_b, part_g);
    } else {
      if (ln)
        hipLaunchKernelGGL((colsum_part_k<float, true>), grid, dim3(NT), 0, s, (const float*)dout, ld,
                           (const float*)x, mean, rstd, rows, n, part_b, part_g);
      else
        hipLaunchKernelGGL((colsum_part_k<float, false>), grid, dim3(NT), 0, s, (const float*)dout,
                           ld, (const float*)nullptr, mean, rstd, rows, n, part_b, part_g);
    }
  }
  dim3 g1((n + NT - 1) / NT);
  hipLaunchKernelGGL(colsum_final_k, g1, dim3(NT), 0, s, (const float*)part_b, nchunk, n, db,
                     accumulate);
  if (ln)
    hipLaunchKernelGGL(colsum_final_k, g1, dim3(NT), 0, s, (const float*)part_g, nchunk, n, dg,
                       accumulate);
  return hipGetLastError();
}

hipError_t colsum_bias(int elt, const void* dout, long ld, long rows, int n, float* db,
                       int accumulate, float* part, hipStream_t s) {
  return colsum_impl(elt, false, dout, ld, nullptr, nullptr, nullptr, rows, n, nullptr, db,
                     accumulate, part, s);
}

hipError_t colsum_ln(int elt, const void* dout, const void* x, const float* mean,
                     const float* rstd, long rows, int n, float* dg, float* db, int accumulate,
                     float* part, hipStream_t s) {
  return colsum_impl(elt, true, dout, n, x, mean, rstd, rows, n, dg, db, accumulate, part, s);
}
