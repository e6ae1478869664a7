// LayerNorm forward / input-gradient kernels (one wave per token row; rows
// too long for one wave take a workgroup), fp32 statistics, wavefront-shuffle
// reductions; and the deterministic column reductions of the weight pass
// (bias and LayerNorm-affine gradients).
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

// Sum of rows [r0, r1) of columns c..c+3 of a [rows][n] fp32 array, in row
// order; rows are requested 8 at a time before they are added, so the loads
// overlap instead of each waiting for the previous sum.
__device__ __forceinline__ float4 sum_rows4(const float* src, int r0, int r1, int n, int c) {
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  int r = r0;
  for (; r + 8 <= r1; r += 8) {
    float4 v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = *(const float4*)(src + (long)(r + i) * n + c);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      s.x += v[i].x; s.y += v[i].y; s.z += v[i].z; s.w += v[i].w;
    }
  }
  for (; r < r1; ++r) {
    const float4 v = *(const float4*)(src + (long)r * n + c);
    s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
  }
  return s;
}

// Middle stage of the column sums: block row g sums partial rows
// [MID g, MID g + MID) in order (a fixed tree: partials -> groups of MID ->
// final); blockIdx.z selects the array (0: the plain sums, 1: the LN-gamma
// sums, stored right after them, as are their groups).
constexpr int MID = 16;
__global__ __launch_bounds__(NT) void colsum_mid_k(const float* __restrict__ part, int nchunk, int n,
                                                   float* __restrict__ mid) {
  const int c = 4 * (blockIdx.x * NT + threadIdx.x);
  if (c >= n) return;
  const float* src = part + (long)blockIdx.z * nchunk * n;
  float* dst = mid + (long)blockIdx.z * gridDim.y * n;
  const int r0 = blockIdx.y * MID, r1 = min(nchunk, r0 + MID);
  *(float4*)(dst + (long)blockIdx.y * n + c) = sum_rows4(src, r0, r1, n, c);
}

// Last stage: rows [0, nchunk) into out_b (blockIdx.y = 0) or rows
// [nchunk, 2 nchunk) into out_g (blockIdx.y = 1), in order.
__global__ __launch_bounds__(NT) void colsum_final_k(const float* __restrict__ part, int nchunk, int n,
                                                     float* __restrict__ out_b, float* __restrict__ out_g,
                                                     int accumulate) {
  const int c = 4 * (blockIdx.x * NT + threadIdx.x);
  if (c >= n) return;
  const float* src = part + (long)blockIdx.y * nchunk * n;
  float4 s = sum_rows4(src, 0, nchunk, n, c);
  float4* o = (float4*)((blockIdx.y ? out_g : out_b) + c);
  if (accumulate) {
    const float4 v = *o;
    s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
  }
  *o = s;
}

// ---------------------------------------------------------------------------
// One wave per row with the row held in registers as 16-byte chunks (one HBM
// pass per tensor; MAXC chunks per lane cover rows of up to 64 * MAXC chunks).
template <class E>
struct Chunk {
  static constexpr int N = 16 / sizeof(E);  // elements per 16-byte chunk
};

__device__ __forceinline__ void unpack(const uint4& u, const bf16*, float (&f)[8]) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void unpack(const uint4& u, const float*, float (&f)[4]) {
  f[0] = __uint_as_float(u.x);
  f[1] = __uint_as_float(u.y);
  f[2] = __uint_as_float(u.z);
  f[3] = __uint_as_float(u.w);
}
__device__ __forceinline__ uint4 pack(const float (&f)[8], const bf16*) {
  bf16 t[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) t[i] = (bf16)f[i];
  return *(const uint4*)t;
}
__device__ __forceinline__ uint4 pack(const float (&f)[4], const float*) {
  return make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]),
                    __float_as_uint(f[3]));
}

template <class E, int MAXC>
__global__ __launch_bounds__(NT) void ln_fwd_wave_k(const E* __restrict__ x, const float* __restrict__ g,
                                                    const float* __restrict__ b, E* __restrict__ y,
                                                    E* __restrict__ xcopy, float* __restrict__ mean,
                                                    float* __restrict__ rstd, long rows, int h, float eps) {
  constexpr int EPC = Chunk<E>::N;
  const long row = blockIdx.x * (long)(NT / 64) + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int lane = threadIdx.x & 63, nc = h / EPC;
  const E* xr = x + row * h;
  uint4 v[MAXC];
  // For rows of up to 8 chunks per lane gamma and beta are requested with the
  // row, not after its reductions (one wave per row and a single round of
  // waves: a later request adds a whole memory round trip to the kernel);
  // longer rows have no registers to spare for them.
  constexpr bool PRE = MAXC <= 8;
  float gg[PRE ? MAXC : 1][EPC], bb[PRE ? MAXC : 1][EPC];
  auto ld_gb = [&](int q, int c, float (&gq)[EPC], float (&bq)[EPC]) {
#pragma unroll
    for (int e = 0; e < EPC; e += 4) {
      *(float4*)(gq + e) = *(const float4*)(g + (long)c * EPC + e);
      *(float4*)(bq + e) = *(const float4*)(b + (long)c * EPC + e);
    }
  };
#pragma unroll
  for (int q = 0; q < MAXC; ++q) {
    const int c = lane + 64 * q;
    if (c < nc) {
      v[q] = *(const uint4*)(xr + (long)c * EPC);
      if constexpr (PRE) ld_gb(q, c, gg[q], bb[q]);
    }
  }
  float s = 0.f;
#pragma unroll
  for (int q = 0; q < MAXC; ++q) {
    if (lane + 64 * q < nc) {
      float f[EPC];
      unpack(v[q], (const E*)nullptr, f);
#pragma unroll
      for (int e = 0; e < EPC; ++e) s += f[e];
    }
  }
  const float mu = wave_sum(s) / h;
  float qv = 0.f;
#pragma unroll
  for (int q = 0; q < MAXC; ++q) {
    if (lane + 64 * q < nc) {
      float f[EPC];
      unpack(v[q], (const E*)nullptr, f);
#pragma unroll
      for (int e = 0; e < EPC; ++e) qv += (f[e] - mu) * (f[e] - mu);
    }
  }
  const float rs = 1.0f / sqrtf(wave_sum(qv) / h + eps);
  E* yr = y + row * h;
#pragma unroll
  for (int q = 0; q < MAXC; ++q) {
    const int c = lane + 64 * q;
    if (c < nc) {
      float f[EPC];
      unpack(v[q], (const E*)nullptr, f);
      const int qi = PRE ? q : 0;
      if constexpr (!PRE) ld_gb(q, c, gg[0], bb[0]);
#pragma unroll
      for (int e = 0; e < EPC; ++e) f[e] = (f[e] - mu) * rs * gg[qi][e] + bb[qi][e];
      *(uint4*)(yr + (long)c * EPC) = pack(f, (const E*)nullptr);
      if (xcopy) *(uint4*)(xcopy + row * h + (long)c * EPC) = v[q];  // the input row, unchanged
    }
  }
  if (lane == 0) {
    mean[row] = mu;
    rstd[row] = rs;
  }
}

template <class E, int MAXC>
__global__ __launch_bounds__(NT) void ln_bwd_wave_k(const E* __restrict__ dout, const E* __restrict__ x,
                                                    const float* __restrict__ mean,
                                                    const float* __restrict__ rstd,
                                                    const float* __restrict__ g,
                                                    const E* __restrict__ resid, E* __restrict__ dx,
                                                    E* __restrict__ rcopy, long rows, int h) {
  constexpr int EPC = Chunk<E>::N;
  const long row = blockIdx.x * (long)(NT / 64) + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int lane = threadIdx.x & 63, nc = h / EPC;
  const float mu = mean[row], rs = rstd[row];
  // For rows of up to 8 chunks per lane every input of the row (the residual
  // and gamma too) is requested before the reductions, so the kernel pays one
  // memory round trip, not two; longer rows load them where they are used.
  constexpr bool PRE = MAXC <= 8;
  uint4 dv[MAXC], xv[MAXC], rv[PRE ? MAXC : 1];
  float gg[PRE ? MAXC : 1][EPC];
  auto ld_g = [&](int c, float (&gq)[EPC]) {
#pragma unroll
    for (int e = 0; e < EPC; e += 4) *(float4*)(gq + e) = *(const float4*)(g + (long)c * EPC + e);
  };
#pragma unroll
  for (int q = 0; q < MAXC; ++q) {
    const int c = lane + 64 * q;
    if (c < nc) {
      dv[q] = *(const uint4*)(dout + row * h + (long)c * EPC);
      xv[q] = *(const uint4*)(x + row * h + (long)c * EPC);
      if constexpr (PRE) {
        rv[q] = *(const uint4*)(resid + row * h + (long)c * EPC);
        ld_g(c, gg[q]);
      }
    }
  }
  float s1 = 0.f, s2 = 0.f;
#pragma unroll
  for (int q = 0; q < MAXC; ++q) {
    const int c = lane + 64 * q;
    if (c < nc) {
      float d[EPC], xx[EPC];
      unpack(dv[q], (const E*)nullptr, d);
      unpack(xv[q], (const E*)nullptr, xx);
      const int qi = PRE ? q : 0;
      if constexpr (!PRE) ld_g(c, gg[0]);
#pragma unroll
      for (int e = 0; e < EPC; ++e) {
        const float dz = d[e] * gg[qi][e];
        s1 += dz;
        s2 += dz * (xx[e] - mu) * rs;
      }
    }
  }
  const float m1 = wave_sum(s1) / h, m2 = wave_sum(s2) / h;
#pragma unroll
  for (int q = 0; q < MAXC; ++q) {
    const int c = lane + 64 * q;
    if (c < nc) {
      float d[EPC], xx[EPC], r[EPC];
      unpack(dv[q], (const E*)nullptr, d);
      unpack(xv[q], (const E*)nullptr, xx);
      const int qi = PRE ? q : 0;
      uint4 rq;
      if constexpr (PRE) {
        rq = rv[q];
      } else {
        rq = *(const uint4*)(resid + row * h + (long)c * EPC);
        ld_g(c, gg[0]);
      }
      unpack(rq, (const E*)nullptr, r);
      if (rcopy) *(uint4*)(rcopy + row * h + (long)c * EPC) = rq;  // the residual row, unchanged
#pragma unroll
      for (int e = 0; e < EPC; ++e) {
        const float xh = (xx[e] - mu) * rs;
        r[e] += rs * (d[e] * gg[qi][e] - m1 - xh * m2);
      }
      *(uint4*)(dx + row * h + (long)c * EPC) = pack(r, (const E*)nullptr);
    }
  }
}

// Column sums with 16-byte loads: thread = one 16-byte column chunk, block
// row y = (segment, 64-row chunk); rows unrolled by 8 for loads in flight.
template <class E, bool LN>
__global__ __launch_bounds__(NT) void colsum_part16_k(ColSegs sg, long ld, long rows, int n, int cps,
                                                      float* __restrict__ part_b,
                                                      float* __restrict__ part_g) {
  constexpr int EPC = Chunk<E>::N;
  const int c = EPC * (blockIdx.x * NT + threadIdx.x);
  if (c >= n) return;
  const int seg = blockIdx.y / cps, ch = blockIdx.y % cps;
  const E* dout = (const E*)sg.dout[seg];
  const E* x = (const E*)sg.x[seg];
  const float* mean = sg.mean[seg];
  const float* rstd = sg.rstd[seg];
  const long r0 = (long)ch * CHUNK;
  const int nr = (int)min((long)CHUNK, rows - r0);
  float sb[EPC], sgm[EPC];
#pragma unroll
  for (int e = 0; e < EPC; ++e) sb[e] = sgm[e] = 0.f;
  for (int r = 0; r < nr; r += 8) {
    uint4 dvv[8], xvv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (r + u < nr) {
        dvv[u] = *(const uint4*)(dout + (r0 + r + u) * ld + c);
        if (LN) xvv[u] = *(const uint4*)(x + (r0 + r + u) * n + c);
      }
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (r + u < nr) {
        float d[EPC];
        unpack(dvv[u], (const E*)nullptr, d);
#pragma unroll
        for (int e = 0; e < EPC; ++e) sb[e] += d[e];
        if (LN) {
          float xx[EPC];
          unpack(xvv[u], (const E*)nullptr, xx);
          const float mu = mean[r0 + r + u], rs = rstd[r0 + r + u];
#pragma unroll
          for (int e = 0; e < EPC; ++e) sgm[e] += d[e] * (xx[e] - mu) * rs;
        }
      }
  }
#pragma unroll
  for (int e = 0; e < EPC; e += 4) {
    *(float4*)(part_b + (long)blockIdx.y * n + c + e) = make_float4(sb[e], sb[e + 1], sb[e + 2], sb[e + 3]);
    if (LN)
      *(float4*)(part_g + (long)blockIdx.y * n + c + e) =
          make_float4(sgm[e], sgm[e + 1], sgm[e + 2], sgm[e + 3]);
  }
}

template <class E, int MAXC>
void launch_ln_fwd(const void* x, const float* g, const float* b, void* y, void* xcopy, float* mean,
                   float* rstd, long rows, int h, float eps, hipStream_t s) {
  hipLaunchKernelGGL((ln_fwd_wave_k<E, MAXC>), dim3((unsigned)((rows + 3) / 4)), dim3(NT), 0, s,
                     (const E*)x, g, b, (E*)y, (E*)xcopy, mean, rstd, rows, h, eps);
}
template <class E, int MAXC>
void launch_ln_bwd(const void* dout, const void* x, const float* mean, const float* rstd, const float* g,
                   const void* resid, void* dx, void* rcopy, long rows, int h, hipStream_t s) {
  hipLaunchKernelGGL((ln_bwd_wave_k<E, MAXC>), dim3((unsigned)((rows + 3) / 4)), dim3(NT), 0, s,
                     (const E*)dout, (const E*)x, mean, rstd, g, (const E*)resid, (E*)dx, (E*)rcopy, rows,
                     h);
}

// chunks per lane of a row of h elements of type E, or 0 when the wave
// kernels do not apply (h not a multiple of the chunk, or too long)
int wave_chunks(int elt, int h) {
  const int epc = 16 / elt;
  if (h % epc) return 0;
  const int per = (h / epc + 63) / 64;
  return per <= 24 ? per : 0;
}

}  // namespace

hipError_t ln_forward(int elt, const void* x, const float* g, const float* b, void* y, float* mean,
                      float* rstd, long rows, int h, float eps, hipStream_t s, void* xcopy) {
  if (rows <= 0) return hipSuccess;
  if (const int per = wave_chunks(elt, h)) {
    if (elt == 2) {
      if (per <= 4) launch_ln_fwd<bf16, 4>(x, g, b, y, xcopy, mean, rstd, rows, h, eps, s);
      else if (per <= 8) launch_ln_fwd<bf16, 8>(x, g, b, y, xcopy, mean, rstd, rows, h, eps, s);
      else if (per <= 12) launch_ln_fwd<bf16, 12>(x, g, b, y, xcopy, mean, rstd, rows, h, eps, s);
      else launch_ln_fwd<bf16, 24>(x, g, b, y, xcopy, mean, rstd, rows, h, eps, s);
    } else {
      if (per <= 4) launch_ln_fwd<float, 4>(x, g, b, y, xcopy, mean, rstd, rows, h, eps, s);
      else if (per <= 8) launch_ln_fwd<float, 8>(x, g, b, y, xcopy, mean, rstd, rows, h, eps, s);
      else launch_ln_fwd<float, 24>(x, g, b, y, xcopy, mean, rstd, rows, h, eps, s);
    }
    return hipGetLastError();
  }
  if (xcopy) {  // the row-per-workgroup kernel writes y only
    const hipError_t e = hipMemcpyAsync(xcopy, x, (size_t)rows * h * elt, hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return e;
  }
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
                       int h, hipStream_t s, void* rcopy) {
  if (rows <= 0) return hipSuccess;
  if (const int per = wave_chunks(elt, h)) {
    if (elt == 2) {
      if (per <= 4) launch_ln_bwd<bf16, 4>(dout, x, mean, rstd, g, resid, dx, rcopy, rows, h, s);
      else if (per <= 8) launch_ln_bwd<bf16, 8>(dout, x, mean, rstd, g, resid, dx, rcopy, rows, h, s);
      else if (per <= 12) launch_ln_bwd<bf16, 12>(dout, x, mean, rstd, g, resid, dx, rcopy, rows, h, s);
      else launch_ln_bwd<bf16, 24>(dout, x, mean, rstd, g, resid, dx, rcopy, rows, h, s);
    } else {
      if (per <= 4) launch_ln_bwd<float, 4>(dout, x, mean, rstd, g, resid, dx, rcopy, rows, h, s);
      else if (per <= 8) launch_ln_bwd<float, 8>(dout, x, mean, rstd, g, resid, dx, rcopy, rows, h, s);
      else launch_ln_bwd<float, 24>(dout, x, mean, rstd, g, resid, dx, rcopy, rows, h, s);
    }
    return hipGetLastError();
  }
  if (rcopy) {  // the row-per-workgroup kernel writes dx only
    const hipError_t e = hipMemcpyAsync(rcopy, resid, (size_t)rows * h * elt, hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return e;
  }
  if (elt == 2)
    hipLaunchKernelGGL(ln_bwd_k<bf16>, dim3(rows), dim3(NT), 0, s, (const bf16*)dout, (const bf16*)x,
                       mean, rstd, g, (const bf16*)resid, (bf16*)dx, h);
  else
    hipLaunchKernelGGL(ln_bwd_k<float>, dim3(rows), dim3(NT), 0, s, (const float*)dout,
                       (const float*)x, mean, rstd, g, (const float*)resid, (float*)dx, h);
  return hipGetLastError();
}

long colsum_part_floats(long rows, int n, int nseg) {
  const long nchunk = nseg * ((rows + CHUNK - 1) / CHUNK);
  return 2 * (nchunk + (nchunk + MID - 1) / MID) * (long)n;
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
  const int epc = 16 / elt;
  if (nchunk > 0 && n % epc == 0 && ld % epc == 0) {
    dim3 grid((n / epc + NT - 1) / NT, nchunk);
    if (elt == 2) {
      if (ln)
        hipLaunchKernelGGL((colsum_part16_k<bf16, true>), grid, dim3(NT), 0, s, sg, ld, rows, n, cps, part_b, part_g);
      else
        hipLaunchKernelGGL((colsum_part16_k<bf16, false>), grid, dim3(NT), 0, s, sg, ld, rows, n, cps, part_b, part_g);
    } else {
      if (ln)
        hipLaunchKernelGGL((colsum_part16_k<float, true>), grid, dim3(NT), 0, s, sg, ld, rows, n, cps, part_b, part_g);
      else
        hipLaunchKernelGGL((colsum_part16_k<float, false>), grid, dim3(NT), 0, s, sg, ld, rows, n, cps, part_b, part_g);
    }
  } else if (nchunk > 0) {
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
  // partial rows -> groups of MID (wide grid) -> one row per column; the plain
  // and (LN) gamma arrays share each launch
  const int narr = ln ? 2 : 1;
  const float* fin = part_b;  // the gamma rows follow the plain ones at every stage
  int nfin = nchunk;
  if (nchunk > MID) {
    const int ng = (nchunk + MID - 1) / MID;
    float* mid = part + 2L * nchunk * n;
    hipLaunchKernelGGL(colsum_mid_k, dim3(cb, ng, narr), dim3(NT), 0, s, (const float*)part_b, nchunk, n, mid);
    fin = mid;
    nfin = ng;
  }
  hipLaunchKernelGGL(colsum_final_k, dim3(cb, narr), dim3(NT), 0, s, fin, nfin, n, db, dg, accumulate);
  return hipGetLastError();
}
