// bf16 GEMM kernel template on CDNA4 matrix cores: v_mfma_f32_32x32x16_bf16, fp32 accumulate.
//
// Workgroup: 256 threads = 4 waves in a 2x2 grid; block tile BM x BN x 64,
// each wave owns (BM/2) x (BN/2) = TM x TN MFMA blocks of 32x32.
// Operands are staged in LDS as [rows][64] k-contiguous tiles (16-byte chunks
// XOR-swizzled so that fragment reads and tile writes spread over the banks),
// double buffered: the global loads of k-tile t+1 are in flight while the
// MFMAs of tile t run, with one barrier per k-tile.
// An operand that is contiguous along M/N in memory (the reduction over
// tokens of the weight-gradient GEMMs, the weights [in, out] of the forward)
// is read in 16-byte vectors along M/N and transposed 8x8 in registers before
// the LDS write, so the MFMA fragments are always k-contiguous.
#pragma once
#include "gemm.h"

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

namespace {

constexpr int BK = 64;
constexpr int NT = 256;

__device__ __forceinline__ int swz(int r) { return ((r >> 1) ^ (r >> 3)) & 7; }

// Element offset of the 8-element chunk c of row r in a [rows][64] tile.
__device__ __forceinline__ int lds_off(int r, int c) { return r * BK + ((c ^ swz(r)) << 3); }

// Rows of an operand tile read from a k-contiguous matrix: row r = mn0 + r,
// element (r, k) at base[(mn0 + r) * ld + k].
template <int ROWS>
struct LoadK {
  static constexpr int NV = ROWS * 8 / NT;
  uint4 v[NV];
  __device__ __forceinline__ void load(const bf16* __restrict__ base, long ld, int mn0, int MN,
                                       int k0, int K) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int idx = threadIdx.x + i * NT;
      const int r = idx >> 3, c = idx & 7;
      const int mn = mn0 + r, k = k0 + c * 8;
      if (mn < MN && k < K)
        v[i] = *(const uint4*)(base + (long)mn * ld + k);
      else
        v[i] = make_uint4(0, 0, 0, 0);
    }
  }
  __device__ __forceinline__ void store(bf16* s) const {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int idx = threadIdx.x + i * NT;
      const int r = idx >> 3, c = idx & 7;
      *(uint4*)(s + lds_off(r, c)) = v[i];
    }
  }
};

__device__ __forceinline__ uint32_t comp(const uint4& u, int i) {
  return i == 0 ? u.x : (i == 1 ? u.y : (i == 2 ? u.z : u.w));
}

// Rows of an operand tile read from an mn-contiguous matrix: element (r, k)
// at base[k * ld + mn0 + r].  Each thread owns 8x8 blocks (8 k x 8 mn).
template <int ROWS>
struct LoadMN {
  static constexpr int NBLK = ROWS;              // (64 / 8) * (ROWS / 8)
  static constexpr int NB = NBLK >= NT ? NBLK / NT : 1;
  uint4 v[NB][8];
  __device__ __forceinline__ void load(const bf16* __restrict__ base, long ld, int mn0, int MN,
                                       int k0, int K) {
#pragma unroll
    for (int bi = 0; bi < NB; ++bi) {
      const int b = threadIdx.x + bi * NT;
      const int mb = b % (ROWS / 8), kb = b / (ROWS / 8);
      const int mn = mn0 + mb * 8;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const int k = k0 + kb * 8 + r;
        if (b < NBLK && mn < MN && k < K)
          v[bi][r] = *(const uint4*)(base + (long)k * ld + mn);
        else
          v[bi][r] = make_uint4(0, 0, 0, 0);
      }
    }
  }
  __device__ __forceinline__ void store(bf16* s) const {
#pragma unroll
    for (int bi = 0; bi < NB; ++bi) {
      const int b = threadIdx.x + bi * NT;
      if (b >= NBLK) continue;
      const int mb = b % (ROWS / 8), kb = b / (ROWS / 8);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        uint32_t o[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t x = comp(v[bi][2 * q], j >> 1), y = comp(v[bi][2 * q + 1], j >> 1);
          o[q] = (j & 1) ? ((x >> 16) | (y & 0xFFFF0000u)) : ((x & 0xFFFFu) | (y << 16));
        }
        *(uint4*)(s + lds_off(mb * 8 + j, kb)) = make_uint4(o[0], o[1], o[2], o[3]);
      }
    }
  }
};

template <int ROWS, bool KC> struct Loader;
template <int ROWS> struct Loader<ROWS, true> : LoadK<ROWS> {};
template <int ROWS> struct Loader<ROWS, false> : LoadMN<ROWS> {};

template <int BM, int BN, int TM, int TN, int EPI>
__device__ __forceinline__ void epilogue(const GemmParams& p, f32x16 (&acc)[TM][TN], int m0, int n0,
                                         int wm, int wn, int lane, long c_off) {
  typedef typename EpiOut<EPI, bf16>::type OutT;
  OutT* C = (OutT*)p.C + c_off;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = n0 + wn * (BN / 2) + j * 32 + (lane & 31);
      if (n >= p.N) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * (BM / 2) + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (m < p.M) epi_store<EPI, bf16>(p, (bf16*)C, m, n, acc[i][j][r]);
      }
    }
}

template <int BM, int BN, bool AK, bool BKC, int EPI>
__global__ __launch_bounds__(NT) void gemm_bf16_kernel(GemmParams p) {
  constexpr int TM = BM / 64, TN = BN / 64;  // 32x32 blocks per wave (wave tile = BM/2 x BN/2)
  __shared__ __attribute__((aligned(16))) bf16 sA[2][BM * BK];
  __shared__ __attribute__((aligned(16))) bf16 sB[2][BN * BK];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // Tile order: spread consecutive tiles over the 8 XCDs' own ranges, then
  // group tile-rows so concurrently running tiles share operand panels in L2.
  const int tiles_m = (p.M + BM - 1) / BM, tiles_n = (p.N + BN - 1) / BN;
  int pid = blockIdx.x;
  const int ntiles = gridDim.x;
  if ((ntiles & 7) == 0) pid = (pid & 7) * (ntiles >> 3) + (pid >> 3);
  constexpr int GM = 8;
  const int width = GM * tiles_n;
  const int first_m = (pid / width) * GM;
  const int gsz = min(tiles_m - first_m, GM);
  const int tm = first_m + (pid % width) % gsz;
  const int tn = (pid % width) / gsz;
  const int m0 = tm * BM, n0 = tn * BN;
  if (p.causal_skip && n0 > m0 + BM - 1) return;

  const int z = blockIdx.y;
  const int zb = z / p.heads, zh = z % p.heads;
  const bf16* A = (const bf16*)p.A + zb * p.a_bs + zh * p.a_hs;
  const bf16* B = (const bf16*)p.B + zb * p.b_bs + zh * p.b_hs;
  const long c_off = zb * p.c_bs + zh * p.c_hs;

  int kb = 0, ke = p.K;
  if (p.krange == KR_BELOW) ke = min(p.K, m0 + BM);
  else if (p.krange == KR_ABOVE) kb = (m0 / BK) * BK;
  const int nk = ke > kb ? (ke - kb + BK - 1) / BK : 0;

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  Loader<BM, AK> la;
  Loader<BN, BKC> lb;
  if (nk > 0) {
    la.load(A, p.lda, m0, p.M, kb, ke);
    lb.load(B, p.ldb, n0, p.N, kb, ke);
    la.store(sA[0]);
    lb.store(sB[0]);
  }
  __syncthreads();

  for (int t = 0; t < nk; ++t) {
    const int cur = t & 1;
    const bool more = t + 1 < nk;
    if (more) {
      la.load(A, p.lda, m0, p.M, kb + (t + 1) * BK, ke);
      lb.load(B, p.ldb, n0, p.N, kb + (t + 1) * BK, ke);
    }
    const bf16* a_s = sA[cur];
    const bf16* b_s = sB[cur];
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int c = ks * 2 + (lane >> 5);
      bf16x8 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *(const bf16x8*)(a_s + lds_off(wm * (BM / 2) + i * 32 + (lane & 31), c));
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = *(const bf16x8*)(b_s + lds_off(wn * (BN / 2) + j * 32 + (lane & 31), c));
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
      la.store(sA[cur ^ 1]);
      lb.store(sB[cur ^ 1]);
    }
    __syncthreads();
  }

  epilogue<BM, BN, TM, TN, EPI>(p, acc, m0, n0, wm, wn, lane, c_off);
}

template <bool AK, bool BKC, int EPI>
hipError_t launch_bf16(const GemmParams& p, hipStream_t s) {
  const long z = (long)p.batch * p.heads;
  auto cost = [&](int bm, int bn) {
    long t = (long)((p.M + bm - 1) / bm) * ((p.N + bn - 1) / bn) * z;
    return ((t + 255) / 256) * (long)bm * bn;
  };
  // Tile choice: the fewest (waves of 256 workgroups) x (tile area), i.e. the
  // least padded work on 256 compute units; ties go to the larger tile, which
  // re-reads its operands less.
  if (p.N <= 128 || cost(256, 128) < cost(256, 256)) {
    const int tiles = ((p.M + 255) / 256) * ((p.N + 127) / 128);
    hipLaunchKernelGGL((gemm_bf16_kernel<256, 128, AK, BKC, EPI>), dim3(tiles, z), dim3(NT), 0, s, p);
  } else {
    const int tiles = ((p.M + 255) / 256) * ((p.N + 255) / 256);
    hipLaunchKernelGGL((gemm_bf16_kernel<256, 256, AK, BKC, EPI>), dim3(tiles, z), dim3(NT), 0, s, p);
  }
  return hipGetLastError();
}

}  // namespace
