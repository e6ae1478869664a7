// GEMM entry points used by the stage runtime, and the shared epilogue.
//
// C[m, n] = sum_k A(m, k) B(k, n) with
//   A(m, k) = a_kcontig ? A[m*lda + k] : A[k*lda + m]
//   B(k, n) = b_kcontig ? B[n*ldb + k] : B[k*ldb + n]
// so every operand layout of the stage maps onto one kernel family:
//   forward  Y  = X W      : A k-contiguous, B n-contiguous (W stored [in, out])
//   dgrad    dX = dY W^T   : A k-contiguous, B k-contiguous
//   wgrad    dW = X^T dY   : A m-contiguous, B n-contiguous (reduction over tokens)
// Optional batching over z = blockIdx.y in [0, batch*heads) adds
// (z / heads) * *_bs + (z % heads) * *_hs elements to A, B and C (attention).
#pragma once

#include <hip/hip_runtime.h>

#include "common.h"

enum EpiKind {
  EPI_STORE = 0,       // C = acc                                (activation type)
  EPI_BIAS = 1,        // C = acc + bias[n]
  EPI_BIAS_RESID = 2,  // C = acc + bias[n] + resid[m, n]
  EPI_BIAS_GELU = 3,   // u = acc + bias[n];  C = gelu'(u), C2 = gelu(u)
  EPI_GELU_BWD = 4,    // C = acc * aux[m, n]   (aux: the stored gelu'(u))
  EPI_F32_ACC = 5,     // C32 = (accumulate ? C32 : 0) + acc     (fp32 gradient buffers)
  EPI_F32_STORE = 6    // C32 = acc                              (fp32 scores)
};

enum KRange {
  KR_FULL = 0,   // k in [0, K)
  KR_BELOW = 1,  // k < min(K, m0 + BM): operand A is zero for k > m (causal P, dS)
  KR_ABOVE = 2   // k >= m0 rounded down: operand A is zero for k < m (transposed causal P, dS)
};

constexpr int GEMM_MAX_SEG = 32;

struct GemmParams {
  int M, N, K;
  const void* A; long lda; int a_kcontig;
  const void* B; long ldb; int b_kcontig;
  int batch, heads;
  long a_bs, a_hs, b_bs, b_hs, c_bs, c_hs;
  int causal_skip;  // skip output tiles strictly above the diagonal (n0 > m0 + BM - 1)
  int krange;       // KRange
  int epi;          // EpiKind
  void* C; long ldc;
  const float* bias;
  const void* resid; long ld_resid;
  const void* aux; long ld_aux;
  void* C2; long ldc2;
  int accumulate;
  // Column sums of B over k (bf16 GEMMs with A and B m/n-contiguous): the
  // bias gradient of a linear layer is exactly this sum of its output
  // gradient, the B operand of its weight-gradient product.  The workgroup of
  // tile-row tm sums the B tiles it stages anyway whose k-tile index t has
  // t mod tiles_m == tm, into row tm of colsum_work (gemm_colsum_floats
  // floats); a second kernel adds the rows in a fixed order and writes
  // (colsum_acc: adds) them to colsum_out[0, N) in fp32.  nullptr: off.
  float* colsum_out;
  int colsum_acc;
  float* colsum_work;
  // Reduction split into segments of kseg_len (0: one segment).  Segment s
  // of A / B starts at segA[s] / segB[s] (A, B are ignored); within a segment
  // the layouts above apply with k counted from the segment start.  Used to
  // run several micro-batches' weight gradients as one product over their
  // concatenated tokens.
  int kseg_len;
  const void* segA[GEMM_MAX_SEG];
  const void* segB[GEMM_MAX_SEG];
};

// Shapes must satisfy: M, N, K multiples of 8 when an operand is loaded
// along that dimension in 8-element vectors (checked by the caller).
hipError_t gemm_bf16(const GemmParams& p, hipStream_t s);
// Floats of colsum_work a bf16 GEMM of M rows and N columns needs (its
// tile-rows are 256 high).
inline long gemm_colsum_floats(long M, long N) { return ((M + 255) / 256) * N; }
hipError_t gemm_f32(const GemmParams& p, hipStream_t s);

template <int EPI, class E>
__device__ __forceinline__ void epi_store(const GemmParams& p, E* C, int m, int n, float v) {
  const long i = (long)m * p.ldc + n;
  if constexpr (EPI == EPI_STORE) {
    C[i] = from_f32<E>(v);
  } else if constexpr (EPI == EPI_BIAS) {
    C[i] = from_f32<E>(v + p.bias[n]);
  } else if constexpr (EPI == EPI_BIAS_RESID) {
    const E* r = (const E*)p.resid;
    C[i] = from_f32<E>(v + p.bias[n] + to_f32(r[(long)m * p.ld_resid + n]));
  } else if constexpr (EPI == EPI_BIAS_GELU) {
    const float u = v + p.bias[n], sg = gelu_sig(u);
    C[i] = from_f32<E>(gelu_grad_s(u, sg));
    ((E*)p.C2)[(long)m * p.ldc2 + n] = from_f32<E>(u * sg);
  } else if constexpr (EPI == EPI_GELU_BWD) {
    const E* d = (const E*)p.aux;
    C[i] = from_f32<E>(v * to_f32(d[(long)m * p.ld_aux + n]));
  } else if constexpr (EPI == EPI_F32_ACC) {
    float* c = (float*)C;
    c[i] = p.accumulate ? c[i] + v : v;
  } else {  // EPI_F32_STORE
    ((float*)C)[i] = v;
  }
}

// Per-element input of an epilogue at (m, n..n+3): the residual, GeLU's
// input, or the fp32 gradient being accumulated into.  Fetched separately
// from the arithmetic so that a tile's epilogue can have a whole block-row of
// these loads in flight instead of one load round trip per output group.
template <int EPI>
struct EpiIn {
  static constexpr bool kHas = EPI == EPI_BIAS_RESID || EPI == EPI_GELU_BWD || EPI == EPI_F32_ACC;
  uint4 raw;
};

template <int EPI, class E>
__device__ __forceinline__ EpiIn<EPI> epi_fetch4(const GemmParams& p, const void* Cv, int m, int n) {
  EpiIn<EPI> r;
  r.raw = make_uint4(0, 0, 0, 0);
  auto ld = [](const E* q) -> uint4 {
    if constexpr (sizeof(E) == 2) {
      const uint2 u = *(const uint2*)q;
      return make_uint4(u.x, u.y, 0, 0);
    } else {
      return *(const uint4*)q;
    }
  };
  if constexpr (EPI == EPI_BIAS_RESID) {
    r.raw = ld((const E*)p.resid + (long)m * p.ld_resid + n);
  } else if constexpr (EPI == EPI_GELU_BWD) {
    r.raw = ld((const E*)p.aux + (long)m * p.ld_aux + n);
  } else if constexpr (EPI == EPI_F32_ACC) {
    if (p.accumulate) r.raw = *(const uint4*)((const float*)Cv + (long)m * p.ldc + n);
  }
  return r;
}

constexpr bool epi_has_bias(int epi) {
  return epi == EPI_BIAS || epi == EPI_BIAS_RESID || epi == EPI_BIAS_GELU;
}

// The epilogue on 4 consecutive columns n..n+3 (n % 4 == 0, all in range)
// given their fetched input and bias[n..n+3] (loaded once by the caller: a
// lane's columns are the same on every row); 8- or 16-byte vector stores.
template <int EPI, class E>
__device__ __forceinline__ void epi_finish4(const GemmParams& p, void* Cv, int m, int n, float4 v,
                                            const EpiIn<EPI>& in, float4 b) {
  const long i = (long)m * p.ldc + n;
  auto cvt4 = [](uint4 u) -> float4 {
    if constexpr (sizeof(E) == 2) {
      return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                         __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
    } else {
      return make_float4(__uint_as_float(u.x), __uint_as_float(u.y), __uint_as_float(u.z),
                         __uint_as_float(u.w));
    }
  };
  auto st4 = [](E* q, float4 f) {
    if constexpr (sizeof(E) == 2) {
      E t[4] = {from_f32<E>(f.x), from_f32<E>(f.y), from_f32<E>(f.z), from_f32<E>(f.w)};
      *(uint2*)q = *(const uint2*)t;
    } else {
      *(float4*)q = f;
    }
  };
  if constexpr (EPI == EPI_F32_ACC) {
    if (p.accumulate) {
      v.x += __uint_as_float(in.raw.x); v.y += __uint_as_float(in.raw.y);
      v.z += __uint_as_float(in.raw.z); v.w += __uint_as_float(in.raw.w);
    }
    *(float4*)((float*)Cv + i) = v;
  } else if constexpr (EPI == EPI_F32_STORE) {
    *(float4*)((float*)Cv + i) = v;
  } else {
    E* C = (E*)Cv;
    if constexpr (epi_has_bias(EPI)) {
      v.x += b.x; v.y += b.y; v.z += b.z; v.w += b.w;
    }
    if constexpr (EPI == EPI_BIAS_RESID) {
      const float4 r = cvt4(in.raw);
      v.x += r.x; v.y += r.y; v.z += r.z; v.w += r.w;
    }
    if constexpr (EPI == EPI_GELU_BWD) {
      const float4 d = cvt4(in.raw);
      v.x *= d.x; v.y *= d.y; v.z *= d.z; v.w *= d.w;
    }
    if constexpr (EPI == EPI_BIAS_GELU) {
      const float4 sg = make_float4(gelu_sig(v.x), gelu_sig(v.y), gelu_sig(v.z), gelu_sig(v.w));
      st4(C + i, make_float4(gelu_grad_s(v.x, sg.x), gelu_grad_s(v.y, sg.y), gelu_grad_s(v.z, sg.z),
                             gelu_grad_s(v.w, sg.w)));
      st4((E*)p.C2 + (long)m * p.ldc2 + n, make_float4(v.x * sg.x, v.y * sg.y, v.z * sg.z, v.w * sg.w));
    } else {
      st4(C + i, v);
    }
  }
}

// Output element type of each epilogue given the activation type E.
template <int EPI, class E>
struct EpiOut { typedef E type; };
template <class E> struct EpiOut<EPI_F32_ACC, E> { typedef float type; };
template <class E> struct EpiOut<EPI_F32_STORE, E> { typedef float type; };
