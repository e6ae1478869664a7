// LayerNorm forward / input-gradient kernels (one workgroup per token row,
// fp32 statistics, wavefront-shuffle reductions) and the deterministic
// column reductions of the weight pass (bias and LayerNorm-affine gradients).
#include "common.h"
#include "kernels.h"

namespace {

constexpr int NT = 256;
constexpr int CHUNK = 64;  // rows per partial sum of the column reductions

__device__ __forceinline__ float4 load4(const float* p) { return *(const float4*)p; }
__device__ __forceinline__ float4 load4(const bf16* p) {
  const uint2 u = *(const uint2*)p;
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                     __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
}

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

// Column sums over the rows of nseg segments (one per micro-batch) of a
// [rows, n] matrix: chunk y of 64 rows of segment y / cps writes its partial
// sums of 4 consecutive columns per thread to part[y][n].
template <class E, bool LN>
__global__ __launch_bounds__(NT) void colsum_part_k(ColSegs sg, long ld, long rows, int n, int cps,
                                                    float* __restrict__ part_b,
                                                    float* __restrict__ part_g) {
  const int c = 4 * (blockIdx.x * NT + threadIdx.x);
  if (c >= n) return;
  const int seg = blockIdx.y / cps, ch = blockIdx.y % cps;
  const E* dout = (const E*)sg.dout[seg];
  const E* x = (const E*)sg.x[seg];
  const float* mean = sg.mean[seg];
  const float* rstd = sg.rstd[seg];
  const long r0 = (long)ch * CHUNK;
  const long r1 = min(rows, r0 + CHUNK);
  float4 sb = make_float4(0.f, 0.f, 0.f, 0.f), sgm = sb;
  for (long r = r0; r < r1; ++r) {
    const float4 d = load4(dout + r * ld + c);
    sb.x += d.x; sb.y += d.y; sb.z += d.z; sb.w += d.w;
    if (LN) {
      const float4 xv = load4(x + r * n + c);
      const float mu = mean[r], rs = rstd[r];
      sgm.x += d.x * (xv.x - mu) * rs;
      sgm.y += d.y * (xv.y - mu) * rs;
      sgm.z += d.z * (xv.z - mu) * rs;
      sgm.w += d.w * (xv.w - mu) * rs;
    }
  }
  *(float4*)(part_b + (long)blockIdx.y * n + c) = sb;
  if (LN) *(float4*)(part_g + (long)blockIdx.y * n + c) = sgm;
}

__global__ __launch_bounds__(NT) void colsum_final_k(const float* __restrict__ part, int nchunk,
                                                     int n, float* __restrict__ out, int accumulate) {
  const int c = 4 * (blockIdx.x * NT + threadIdx.x);
  if (c >= n) return;
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int ch = 0; ch < nchunk; ++ch) {
    const float4 v = *(const float4*)(part + (long)ch * n + c);
    s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
  }
  float4* o = (float4*)(out + c);
  if (accumulate) {
    const float4 v = *o;
    s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
  }
  *o = s;
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

long colsum_part_floats(long rows, int n, int nseg) {
  return 2 * nseg * ((rows + CHUNK - 1) / CHUNK) * (long)n;
}

hipError_t colsum(int elt, bool ln, const ColSegs& sg, int nseg, long ld, long rows, int n, float* dg,
                  float* db, int accumulate, float* part, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (n % 4) return hipErrorInvalidValue;
  const int cps = (int)((rows + CHUNK - 1) / CHUNK);
  const int nchunk = nseg * cps;
  float* part_b = part;
  float* part_g = part + (long)nchunk * n;
  const int cb = (n / 4 + NT - 1) / NT;
  if (nchunk > 0) {
    dim3 grid(cb, nchunk);
    if (elt == 2) {
      if (ln)
        hipLaunchKernelGGL((colsum_part_k<bf16, true>), grid, dim3(NT), 0, s, sg, ld, rows, n, cps, part_b, part_g);
      else
        hipLaunchKernelGGL((colsum_part_k<bf16, false>), grid, dim3(NT), 0, s, sg, ld, rows, n, cps, part_b, part_g);
    } else {
      if (ln)
        hipLaunchKernelGGL((colsum_part_k<float, true>), grid, dim3(NT), 0, s, sg, ld, rows, n, cps, part_b, part_g);
      else
        hipLaunchKernelGGL((colsum_part_k<float, false>), grid, dim3(NT), 0, s, sg, ld, rows, n, cps, part_b, part_g);
    }
  }
  hipLaunchKernelGGL(colsum_final_k, dim3(cb), dim3(NT), 0, s, (const float*)part_b, nchunk, n, db, accumulate);
  if (ln)
    hipLaunchKernelGGL(colsum_final_k, dim3(cb), dim3(NT), 0, s, (const float*)part_g, nchunk, n, dg, accumulate);
  return hipGetLastError();
}
