// Fused AdamW over the stage's flat fp32 parameter / gradient / moment
// buffers (coalesced float4 streams), refreshing the bf16 weight copies in
// the same pass; plus small fill / cast helpers.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int NT = 256;

// The update lr m_hat / (sqrt(v_hat) + eps) from the new moments.  Hardware
// square root and reciprocal (1 ulp each; the update is 1e-4 of a weight, so
// their error stays far below fp32 resolution of the weight).  The rollback
// recomputes it with this same function from the same moments, so it
// subtracts exactly what the step added.
__device__ __forceinline__ float adam_update(float m, float v, float eps, float step_size,
                                             float inv_sqrt_bc2) {
  return step_size * m * __builtin_amdgcn_rcpf(__builtin_amdgcn_sqrtf(v) * inv_sqrt_bc2 + eps);
}

__device__ __forceinline__ float adam_one(float p, float g, float& m, float& v, bool decay,
                                          float lr, float b1, float b2, float eps, float wd,
                                          float step_size, float inv_sqrt_bc2, float gs) {
  g *= gs;
  m = b1 * m + (1.f - b1) * g;
  v = b2 * v + (1.f - b2) * g * g;
  if (decay) p *= (1.f - lr * wd);
  return p - adam_update(m, v, eps, step_size, inv_sqrt_bc2);
}

// The fp32 streams are read and written once per step: non-temporal accesses
// keep them from displacing cached data (-1.6 % AdamW time).
typedef float vf4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ float4 ld_nt(const float4* q) {
  const vf4 t = __builtin_nontemporal_load((const vf4*)q);
  return make_float4(t.x, t.y, t.z, t.w);
}
__device__ __forceinline__ void st_nt(float4* q, float4 v) {
  const vf4 t = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(t, (vf4*)q);
}

// bf16 working copy of 4 consecutive weights: one 8-byte store.
__device__ __forceinline__ void store_bf16x4(bf16* o, float4 w) {
  const bf16 t[4] = {(bf16)w.x, (bf16)w.y, (bf16)w.z, (bf16)w.w};
  *(uint2*)o = *(const uint2*)t;
}

// n and n_decay are multiples of 4 (parameter tensors are padded to 64).
__global__ __launch_bounds__(NT) void adamw_k(float4* __restrict__ p, const float4* __restrict__ g,
                                              float4* __restrict__ m, float4* __restrict__ v,
                                              bf16* __restrict__ wb, long n4, long nd4, float lr,
                                              float b1, float b2, float eps, float wd,
                                              float step_size, float inv_sqrt_bc2, float gs) {
  for (long i = blockIdx.x * (long)NT + threadIdx.x; i < n4; i += (long)gridDim.x * NT) {
    float4 pp = ld_nt(p + i), gg = ld_nt(g + i), mm = ld_nt(m + i), vv = ld_nt(v + i);
    const bool dec = i < nd4;
    pp.x = adam_one(pp.x, gg.x, mm.x, vv.x, dec, lr, b1, b2, eps, wd, step_size, inv_sqrt_bc2, gs);
    pp.y = adam_one(pp.y, gg.y, mm.y, vv.y, dec, lr, b1, b2, eps, wd, step_size, inv_sqrt_bc2, gs);
    pp.z = adam_one(pp.z, gg.z, mm.z, vv.z, dec, lr, b1, b2, eps, wd, step_size, inv_sqrt_bc2, gs);
    pp.w = adam_one(pp.w, gg.w, mm.w, vv.w, dec, lr, b1, b2, eps, wd, step_size, inv_sqrt_bc2, gs);
    st_nt(p + i, pp);
    st_nt(m + i, mm);
    st_nt(v + i, vv);
    if (wb != nullptr && dec) store_bf16x4(wb + 4 * i, pp);
  }
}

// Inverse of adam_one for the same step: the stepped p, m, v and the gradient
// of that step give the values before it (each assignment undone in reverse
// order; v is clamped at zero against rounding).  Undoing the first step
// restores the zero initial moments exactly: recomputed ones would hold fp32
// rounding residue, which the next step's m / sqrt(v) would amplify.
__device__ __forceinline__ float adam_undo(float p, float g, float& m, float& v, bool decay,
                                           float lr, float b1, float b2, float eps, float wd,
                                           float step_size, float inv_sqrt_bc2, float gs, bool first) {
  g *= gs;
  p += adam_update(m, v, eps, step_size, inv_sqrt_bc2);
  if (decay) p /= (1.f - lr * wd);
  v = first ? 0.f : fmaxf((v - (1.f - b2) * g * g) / b2, 0.f);
  m = first ? 0.f : (m - (1.f - b1) * g) / b1;
  return p;
}

__global__ __launch_bounds__(NT) void adamw_undo_k(float4* __restrict__ p, const float4* __restrict__ g,
                                                   float4* __restrict__ m, float4* __restrict__ v,
                                                   bf16* __restrict__ wb, long n4, long nd4, float lr,
                                                   float b1, float b2, float eps, float wd,
                                                   float step_size, float inv_sqrt_bc2, float gs,
                                                   int first) {
  for (long i = blockIdx.x * (long)NT + threadIdx.x; i < n4; i += (long)gridDim.x * NT) {
    float4 pp = p[i], gg = g[i], mm = m[i], vv = v[i];
    const bool dec = i < nd4, f = first != 0;
    pp.x = adam_undo(pp.x, gg.x, mm.x, vv.x, dec, lr, b1, b2, eps, wd, step_size, inv_sqrt_bc2, gs, f);
    pp.y = adam_undo(pp.y, gg.y, mm.y, vv.y, dec, lr, b1, b2, eps, wd, step_size, inv_sqrt_bc2, gs, f);
    pp.z = adam_undo(pp.z, gg.z, mm.z, vv.z, dec, lr, b1, b2, eps, wd, step_size, inv_sqrt_bc2, gs, f);
    pp.w = adam_undo(pp.w, gg.w, mm.w, vv.w, dec, lr, b1, b2, eps, wd, step_size, inv_sqrt_bc2, gs, f);
    p[i] = pp;
    m[i] = mm;
    v[i] = vv;
    if (wb != nullptr && dec) store_bf16x4(wb + 4 * i, pp);
  }
}

// Per-block partial sum of squares of the finite entries of gs * g and count
// of non-finite entries; a fixed grid and fixed reduction order make the
// result bitwise reproducible.
__global__ __launch_bounds__(NT) void grad_check_k(const float4* __restrict__ g, long n4, float gs,
                                                   float* __restrict__ part, int* __restrict__ bad) {
  __shared__ float red[NT / 64];
  __shared__ int redi[NT / 64];
  float s = 0.f;
  int nb = 0;
  for (long i = blockIdx.x * (long)NT + threadIdx.x; i < n4; i += (long)gridDim.x * NT) {
    const float4 v = g[i];
    const float e[4] = {gs * v.x, gs * v.y, gs * v.z, gs * v.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (isfinite(e[k]))
        s += e[k] * e[k];
      else
        ++nb;
    }
  }
  const float tot = block_sum<NT>(s, red);
  int c = nb;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, 64);
  if ((threadIdx.x & 63) == 0) redi[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    int t = 0;
    for (int w = 0; w < NT / 64; ++w) t += redi[w];
    part[blockIdx.x] = tot;
    bad[blockIdx.x] = t;
  }
}

__global__ __launch_bounds__(NT) void cast_k(const float* __restrict__ s, bf16* __restrict__ d, long n) {
  for (long i = blockIdx.x * (long)NT + threadIdx.x; i < n; i += (long)gridDim.x * NT) d[i] = (bf16)s[i];
}

__global__ __launch_bounds__(NT) void fill_k(float* __restrict__ d, long n, float v) {
  for (long i = blockIdx.x * (long)NT + threadIdx.x; i < n; i += (long)gridDim.x * NT) d[i] = v;
}

// Grid-stride launches: up to 32768 workgroups (128 per CU); the AdamW
// stream measured 4.84 TB/s with 8192 and 5.07 TB/s with 32768 (a plain
// device copy reaches 5.2 TB/s on MI355X).
int grid_for(long n) {
  long g = (n + NT - 1) / NT;
  return (int)(g < 32768 ? (g > 0 ? g : 1) : 32768);
}

}  // namespace

hipError_t adamw_step(float* p, const float* g, float* m, float* v, void* wb, long n, long n_decay,
                      float lr, float beta1, float beta2, float eps, float wd, float step_size,
                      float inv_sqrt_bc2, float grad_scale, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if ((n & 3) || (n_decay & 3)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(adamw_k, dim3(grid_for(n / 4)), dim3(NT), 0, s, (float4*)p, (const float4*)g,
                     (float4*)m, (float4*)v, (bf16*)wb, n / 4, n_decay / 4, lr, beta1, beta2, eps,
                     wd, step_size, inv_sqrt_bc2, grad_scale);
  return hipGetLastError();
}

hipError_t adamw_undo(float* p, const float* g, float* m, float* v, void* wb, long n, long n_decay,
                      float lr, float beta1, float beta2, float eps, float wd, float step_size,
                      float inv_sqrt_bc2, float grad_scale, int first_step, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if ((n & 3) || (n_decay & 3)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(adamw_undo_k, dim3(grid_for(n / 4)), dim3(NT), 0, s, (float4*)p, (const float4*)g,
                     (float4*)m, (float4*)v, (bf16*)wb, n / 4, n_decay / 4, lr, beta1, beta2, eps,
                     wd, step_size, inv_sqrt_bc2, grad_scale, first_step);
  return hipGetLastError();
}

hipError_t grad_check(const float* g, long n, float grad_scale, float* part, int* bad, hipStream_t s) {
  if (n <= 0 || (n & 3)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(grad_check_k, dim3(GRAD_CHECK_BLOCKS), dim3(NT), 0, s, (const float4*)g, n / 4,
                     grad_scale, part, bad);
  return hipGetLastError();
}

hipError_t cast_f32_to_bf16(const float* src, void* dst, long n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(cast_k, dim3(grid_for(n)), dim3(NT), 0, s, src, (bf16*)dst, n);
  return hipGetLastError();
}

hipError_t fill_f32(float* dst, long n, float value, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_k, dim3(grid_for(n)), dim3(NT), 0, s, dst, n, value);
  return hipGetLastError();
}
