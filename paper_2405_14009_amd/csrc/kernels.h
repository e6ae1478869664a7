// Host-side launchers of the non-GEMM stage kernels.  Every launcher
// enqueues on the given stream and returns hipGetLastError().
#pragma once

#include <hip/hip_runtime.h>

// LayerNorm forward over rows of width h: y = (x - mean) * rstd * g + b;
// mean and rstd (fp32) are saved per row.  elt: 2 = bf16, 4 = fp32.  When
// xcopy is given, x is also copied there (rows x h elements).
hipError_t ln_forward(int elt, const void* x, const float* g, const float* b, void* y, float* mean,
                      float* rstd, long rows, int h, float eps, hipStream_t s, void* xcopy = nullptr);

// LayerNorm input gradient plus residual: dx = resid + rstd * (dz - mean(dz)
// - xhat * mean(dz * xhat)), dz = dout * g, xhat recomputed from x, mean, rstd.
// When rcopy is given, resid is also copied there (rows x h elements).
hipError_t ln_backward(int elt, const void* dout, const void* x, const float* mean,
                       const float* rstd, const float* g, const void* resid, void* dx, long rows,
                       int h, hipStream_t s, void* rcopy = nullptr);

// Column reductions over the rows of nseg segments (one per micro-batch) of
// a [rows, n] matrix with leading dimension ld, into fp32 outputs (overwrite
// or accumulate); deterministic two-stage sums (64-row partials, then a fixed
// order).  n % 4 == 0.
//   bias (ln = false):  db[c] (+)= sum_r dout[r, c]
//   ln   (ln = true):   dg[c] (+)= sum_r dout[r, c] * (x[r, c] - mean[r]) * rstd[r];  db as above
// (x has leading dimension n).  part must hold colsum_part_floats(rows, n, nseg) floats.
constexpr int COLSUM_MAX_SEG = 32;
struct ColSegs {
  const void* dout[COLSUM_MAX_SEG];
  const void* x[COLSUM_MAX_SEG];
  const float* mean[COLSUM_MAX_SEG];
  const float* rstd[COLSUM_MAX_SEG];
};
hipError_t colsum(int elt, bool ln, const ColSegs& segs, int nseg, long ld, long rows, int n, float* dg,
                  float* db, int accumulate, float* part, hipStream_t s);
long colsum_part_floats(long rows, int n, int nseg);

// Attention softmax over materialised scores, rows of length s, z*s rows.
//   forward:  P[r, c] = exp(scale S[r, c] - max) / sum  for c <= q (causal) else 0
//   backward: dS[r, c] = scale * P[r, c] * (dP[r, c] - sum_c' dP P)  (0 where masked)
hipError_t softmax_forward(int elt, const float* S, void* P, long rows, int s, float scale,
                           int causal, hipStream_t st);
hipError_t softmax_backward(int elt, const float* dP, const void* P, void* dS, long rows, int s,
                            float scale, int causal, hipStream_t st);

// Fused attention core (bf16, head dimension 128): per (sequence, head)
// O = softmax(Q K^T / sqrt(128), causal) V without materialising the scores.
// qkv: [b*s, 3h] with column blocks Q | K | V (head j at columns j*128 of each);
// o: [b*s, h]; lse: [b, heads, s] fp32 base-2 log-sum-exp of the scaled scores
// (written by the forward, read by the backward).  The backward writes dQ, dK,
// dV into the three column blocks of dqkv [b*s, 3h]; dv_scratch holds b*heads*s
// floats.  h == heads * 128.
bool attn_flash_supported(int elt, int head_dim);
// Whether causal fused attention over b sequences of s tokens and `heads`
// heads runs the paired kernels (one workgroup per pair of query blocks) on
// the current device, rather than one workgroup per query block.
bool attn_flash_paired(int b, int s, int heads);
hipError_t attn_flash_forward(const void* qkv, void* o, float* lse, int b, int s, int heads, int h,
                              int causal, hipStream_t st);
hipError_t attn_flash_backward(const void* qkv, const void* o, const void* dout, const float* lse,
                               float* dv_scratch, void* dqkv, int b, int s, int heads, int h, int causal,
                               hipStream_t st);

// AdamW over n fp32 parameters; weight decay on indices < n_decay; when wb is
// non-null the first n_decay updated values are also written to it in bf16.
hipError_t adamw_step(float* p, const float* g, float* m, float* v, void* wb, long n, long n_decay,
                      float lr, float beta1, float beta2, float eps, float wd, float step_size,
                      float inv_sqrt_bc2, float grad_scale, hipStream_t s);

// Inverse of adamw_step for the same step number and gradient (rollback);
// first_step != 0 restores the zero initial moments exactly.
hipError_t adamw_undo(float* p, const float* g, float* m, float* v, void* wb, long n, long n_decay,
                      float lr, float beta1, float beta2, float eps, float wd, float step_size,
                      float inv_sqrt_bc2, float grad_scale, int first_step, hipStream_t s);

// Per-block partials over n fp32 gradients (n % 4 == 0): part[b] = sum of
// squares of the finite entries of grad_scale * g, bad[b] = non-finite count,
// for b < GRAD_CHECK_BLOCKS.
constexpr int GRAD_CHECK_BLOCKS = 1024;
hipError_t grad_check(const float* g, long n, float grad_scale, float* part, int* bad, hipStream_t s);

hipError_t cast_f32_to_bf16(const float* src, void* dst, long n, hipStream_t s);
hipError_t fill_f32(float* dst, long n, float value, hipStream_t s);
