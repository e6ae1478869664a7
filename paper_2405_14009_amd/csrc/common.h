// Shared device helpers for the stage kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16;

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }

template <class E> __device__ __forceinline__ E from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }  // round to nearest even

// tanh form of GeLU: 0.5 u (1 + tanh(z)), z = sqrt(2/pi) (u + 0.044715 u^3).
// Evaluated through the identity 0.5 (1 + tanh z) = 1 / (1 + exp(-2 z)),
// which needs one exponential and one reciprocal and has no cancellation.
// The reciprocal is the hardware one (1 ulp; 1 / inf = 0 for large -u).
__device__ __forceinline__ float gelu_sig(float u) {
  const float c = 0.7978845608028654f;
  const float z = c * (u + 0.044715f * u * u * u);
  return __builtin_amdgcn_rcpf(1.0f + __expf(-2.0f * z));
}

__device__ __forceinline__ float gelu_f(float u) { return u * gelu_sig(u); }

// d/du gelu(u) = s + 2 u s (1 - s) z'(u), s = 0.5 (1 + tanh z), given s.
__device__ __forceinline__ float gelu_grad_s(float u, float s) {
  const float c = 0.7978845608028654f;
  return s + 2.0f * u * s * (1.0f - s) * c * (1.0f + 3.0f * 0.044715f * u * u);
}

__device__ __forceinline__ float gelu_grad_f(float u) { return gelu_grad_s(u, gelu_sig(u)); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Sum over a workgroup of NT threads (NT multiple of 64); every thread gets
// the result.  red must hold NT/64 floats; includes the needed barriers.
template <int NT>
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) s += red[i];
  return s;
}

template <int NT>
__device__ __forceinline__ float block_max(float v, float* red) {
  v = wave_max(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float s = red[0];
#pragma unroll
  for (int i = 1; i < NT / 64; ++i) s = fmaxf(s, red[i]);
  return s;
}

// Compute units of the current device (host; cached per device, 256 when the
// query fails).
inline int device_compute_units() {
  static int cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cache[dev] <= 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cache[dev] = n;
  }
  return cache[dev];
}
