// bf16 GEMM kernel template on CDNA4 matrix cores: v_mfma_f32_32x32x16_bf16,
// fp32 accumulate.
//
// Each wave owns a 128 x 64 output tile (4 x 2 MFMA blocks of 32x32, 128
// accumulators); a workgroup tile of BM x BN uses (BM/128) x (BN/64) waves,
// so a 256x256 tile runs 8 waves (two per SIMD, which hide each other's LDS
// and memory latency) and a 256x128 tile 4 waves.
// Operands are staged in LDS as [rows][64] k-contiguous tiles whose 16-byte
// chunks are XOR-swizzled so fragment reads and tile writes spread over the
// banks, double buffered along k with one barrier per 64-wide k-tile:
// global loads of tile t+1 are in flight while the MFMAs of tile t run, and
// within a tile the fragments of the next 16-wide k-step are read from LDS
// while the current step's MFMAs issue.
// Global loads are buffer loads whose out-of-range offsets return zero, so
// ragged edges need no branches.  An operand that is contiguous along M/N in
// memory (the token reduction of the weight-gradient GEMMs, the [in, out]
// weights of the forward) is read in 16-byte vectors along M/N and
// transposed 8x8 in registers before the LDS write, so MFMA fragments are
// always k-contiguous.
#pragma once

#include <type_traits>

#include "gemm.h"

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

namespace {

constexpr int BK = 64;
constexpr uint32_t kOOB = 0x80000000u;  // buffer offset that is always out of range -> loads 0

__device__ __forceinline__ int swz(int r) { return ((r >> 1) ^ (r >> 3)) & 7; }

// Element offset of the 8-element chunk c of row r in a [rows][64] tile.
__device__ __forceinline__ int lds_off(int r, int c) { return r * BK + ((c ^ swz(r)) << 3); }

// Buffer descriptor over [base, base + bytes); base and size are workgroup
// uniform, and are made provably so (readfirstlane) so that the descriptor
// lives in scalar registers.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, long bytes) {
  const long cap = 0x7fffffffL;
  const uint64_t a = (uint64_t)base;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  const int n = __builtin_amdgcn_readfirstlane((int)(bytes < cap ? bytes : cap));
  return __builtin_amdgcn_make_buffer_rsrc((void*)(((uint64_t)hi << 32) | lo), (short)0, n, 0x00020000);
}

__device__ __forceinline__ uint4 bload(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

__device__ __forceinline__ uint32_t comp(const uint4& u, int i) {
  return i == 0 ? u.x : (i == 1 ? u.y : (i == 2 ? u.z : u.w));
}

// Tile of ROWS rows (m or n) x 64 k from a k-contiguous matrix: element
// (r, k) at base[r * ld + k].  Thread t loads 16-byte chunks t, t+NT, ...
template <int ROWS, int NT>
struct LoadK {
  static constexpr int NV = ROWS * 8 / NT;
  static_assert(NV >= 1, "tile too small for the workgroup");
  uint4 v[NV];
  uint32_t row_off[NV];  // byte offset of the row, kOOB when the row is out of range
  __device__ __forceinline__ void init(long ld, int mn0, int MN) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int idx = threadIdx.x + i * NT;
      const int mn = mn0 + (idx >> 3);
      row_off[i] = mn < MN ? (uint32_t)((long)mn * ld * 2) : kOOB;
    }
  }
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, int k0, int K) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int idx = threadIdx.x + i * NT;
      const int k = k0 + (idx & 7) * 8;
      const uint32_t off = (k < K) ? row_off[i] + 2u * k : kOOB;
      v[i] = bload(r, off | (row_off[i] & kOOB));
    }
  }
  __device__ __forceinline__ void store(bf16* s) const {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int idx = threadIdx.x + i * NT;
      *(uint4*)(s + lds_off(idx >> 3, idx & 7)) = v[i];
    }
  }
};

// Tile of ROWS rows (m or n) x 64 k from an mn-contiguous matrix: element
// (r, k) at base[k * ld + r].  A thread owns one 8(k) x 8(mn) block; block b
// goes to thread (b + SHIFT) % NT so that two such operands use disjoint
// threads.
template <int ROWS, int NT, int SHIFT>
struct LoadMN {
  static constexpr int NBLK = ROWS;  // (64 / 8) * (ROWS / 8)
  static_assert(NBLK <= NT, "one 8x8 block per thread");
  uint4 v[8];
  int b;
  uint32_t col_off;  // byte offset of the thread's 8 columns, kOOB when out of range
  __device__ __forceinline__ void init(int mn0, int MN) {
    b = ((int)threadIdx.x + NT - SHIFT) % NT;
    const int mn = mn0 + (b % (ROWS / 8)) * 8;
    col_off = (b < NBLK && mn < MN) ? (uint32_t)(2 * mn) : kOOB;
  }
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, long ld, int k0, int K) {
    if (b >= NBLK) return;
    const int kb = b / (ROWS / 8);
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int k = k0 + kb * 8 + q;
      const uint32_t off = (k < K) ? col_off + (uint32_t)((long)k * ld * 2) : kOOB;
      v[q] = bload(r, off | (col_off & kOOB));
    }
  }
  __device__ __forceinline__ void store(bf16* s) const {
    if (b >= NBLK) return;
    const int mb = b % (ROWS / 8), kb = b / (ROWS / 8);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      uint32_t o[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t x = comp(v[2 * q], j >> 1), y = comp(v[2 * q + 1], j >> 1);
        o[q] = (j & 1) ? ((x >> 16) | (y & 0xFFFF0000u)) : ((x & 0xFFFFu) | (y << 16));
      }
      *(uint4*)(s + lds_off(mb * 8 + j, kb)) = make_uint4(o[0], o[1], o[2], o[3]);
    }
  }
};

template <int ROWS, int NT, bool KC, int SHIFT> struct Operand;
template <int ROWS, int NT, int SHIFT>
struct Operand<ROWS, NT, true, SHIFT> : LoadK<ROWS, NT> {
  __device__ __forceinline__ void init(long ld, int mn0, int MN) { LoadK<ROWS, NT>::init(ld, mn0, MN); }
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, long, int k0, int K) {
    LoadK<ROWS, NT>::load(r, k0, K);
  }
};
template <int ROWS, int NT, int SHIFT>
struct Operand<ROWS, NT, false, SHIFT> : LoadMN<ROWS, NT, SHIFT> {
  __device__ __forceinline__ void init(long, int mn0, int MN) { LoadMN<ROWS, NT, SHIFT>::init(mn0, MN); }
};

// 512-thread staging of a 256x64 A tile and a 256x64 B tile: threads
// [0, 256) load A, [256, 512) load B, so each thread holds one set of eight
// 16-byte vectors (k-contiguous: eight chunks; mn-contiguous: one 8x8 block).
template <bool AK, bool BKC>
struct SplitLoader {
  uint4 v[8];
  uint32_t off;   // k-contiguous: byte offset of row mn0 + lt/8; mn-contiguous: of column mn0 + 8 (lt%32)
  int nvalid;     // k-contiguous: rows of this thread (lt/8 + 32 i) that are in range; else 0/1
  int lt;
  bool isA;
  template <bool KC>
  __device__ __forceinline__ void init_one(long ld, int mn0, int MN) {
    if constexpr (KC) {
      const int mn = mn0 + (lt >> 3);
      off = (uint32_t)((long)mn * ld * 2);
      nvalid = mn < MN ? (MN - mn + 31) / 32 : 0;
    } else {
      const int mn = mn0 + (lt & 31) * 8;
      off = (uint32_t)(2 * mn);
      nvalid = mn < MN ? 1 : 0;
    }
  }
  __device__ __forceinline__ void init(const GemmParams& p, int m0, int n0) {
    // wave-uniform role, so each branch keeps its buffer descriptor in SGPRs
    isA = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) < 4;
    lt = threadIdx.x & 255;
    if (isA) init_one<AK>(p.lda, m0, p.M);
    else init_one<BKC>(p.ldb, n0, p.N);
  }
  template <bool KC>
  __device__ __forceinline__ void load_one(__amdgpu_buffer_rsrc_t r, long ld, int k0, int K) {
    if constexpr (KC) {
      const int k = k0 + (lt & 7) * 8;
      const uint32_t row_step = (uint32_t)(64 * ld);  // 32 rows, in bytes
      const uint32_t base = off + 2u * k;
#pragma unroll
      for (int i = 0; i < 8; ++i)
        v[i] = bload(r, (k < K && i < nvalid) ? base + i * row_step : kOOB);
    } else {
      const int kb = lt >> 5;
      const uint32_t ld2 = (uint32_t)(2 * ld);
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int k = k0 + kb * 8 + q;
        v[q] = bload(r, (k < K && nvalid) ? off + (uint32_t)k * ld2 : kOOB);
      }
    }
  }
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t rb, long lda,
                                       long ldb, int k0, int K) {
    if (isA) load_one<AK>(ra, lda, k0, K);
    else load_one<BKC>(rb, ldb, k0, K);
  }
  template <bool KC>
  __device__ __forceinline__ void store_one(bf16* s) const {
    if constexpr (KC) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int idx = lt + i * 256;
        *(uint4*)(s + lds_off(idx >> 3, idx & 7)) = v[i];
      }
    } else {
      const int mb = lt & 31, kb = lt >> 5;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        uint32_t o[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t x = comp(v[2 * q], j >> 1), y = comp(v[2 * q + 1], j >> 1);
          o[q] = (j & 1) ? ((x >> 16) | (y & 0xFFFF0000u)) : ((x & 0xFFFFu) | (y << 16));
        }
        *(uint4*)(s + lds_off(mb * 8 + j, kb)) = make_uint4(o[0], o[1], o[2], o[3]);
      }
    }
  }
  __device__ __forceinline__ void store(bf16* sa, bf16* sb) const {
    if (isA) store_one<AK>(sa);
    else store_one<BKC>(sb);
  }
};

template <int BM, int BN, int EPI>
__device__ __forceinline__ void epilogue(const GemmParams& p, f32x16 (&acc)[4][2], int m0, int n0,
                                         int wm, int wn, int lane, long c_off) {
  typedef typename EpiOut<EPI, bf16>::type OutT;
  OutT* C = (OutT*)p.C + c_off;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int n = n0 + wn * 64 + j * 32 + (lane & 31);
      if (n >= p.N) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * 128 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (m < p.M) epi_store<EPI, bf16>(p, (bf16*)C, m, n, acc[i][j][r]);
      }
    }
}

template <int BM, int BN, bool AK, bool BKC, int EPI>
__global__ __launch_bounds__((BM / 128) * (BN / 64) * 64) void gemm_bf16_kernel(GemmParams p) {
  constexpr int WN_ = BN / 64;
  constexpr int NT = (BM / 128) * WN_ * 64;
  __shared__ __attribute__((aligned(16))) bf16 sA[2][BM * BK];
  __shared__ __attribute__((aligned(16))) bf16 sB[2][BN * BK];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN_, wn = wave % WN_;

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
  // Extents of the operands (bytes from their base); rows beyond are zero.
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(A, 2L * (AK ? (long)p.M * p.lda : (long)p.K * p.lda));
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(B, 2L * (BKC ? (long)p.N * p.ldb : (long)p.K * p.ldb));

  int kb = 0, ke = p.K;
  if (p.krange == KR_BELOW) ke = min(p.K, m0 + BM);
  else if (p.krange == KR_ABOVE) kb = (m0 / BK) * BK;
  const int nk = ke > kb ? (ke - kb + BK - 1) / BK : 0;

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // Global -> register -> LDS staging of the k-tiles.
  struct Pair {
    Operand<BM, NT, AK, 0> a;
    Operand<BN, NT, BKC, NT / 2> b;
    __device__ __forceinline__ void init(const GemmParams& p, int m0, int n0) {
      a.init(p.lda, m0, p.M);
      b.init(p.ldb, n0, p.N);
    }
    __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t rb, long lda,
                                         long ldb, int k0, int K) {
      a.load(ra, lda, k0, K);
      b.load(rb, ldb, k0, K);
    }
    __device__ __forceinline__ void store(bf16* sa, bf16* sb) const {
      a.store(sa);
      b.store(sb);
    }
  };
  typedef typename std::conditional<NT == 512 && BM == 256 && BN == 256, SplitLoader<AK, BKC>, Pair>::type Stager;
  Stager ld;
  ld.init(p, m0, n0);
  if (nk > 0) {
    ld.load(ra, rb, p.lda, p.ldb, kb, ke);
    ld.store(sA[0], sB[0]);
  }
  __syncthreads();

  const int arow = wm * 128 + (lane & 31);
  const int brow = wn * 64 + (lane & 31);
  const int chalf = lane >> 5;
  for (int t = 0; t < nk; ++t) {
    const int cur = t & 1;
    const bool more = t + 1 < nk;
    if (more) ld.load(ra, rb, p.lda, p.ldb, kb + (t + 1) * BK, ke);
    const bf16* a_s = sA[cur];
    const bf16* b_s = sB[cur];
    bf16x8 af[2][4], bfr[2][2];
#pragma unroll
    for (int i = 0; i < 4; ++i) af[0][i] = *(const bf16x8*)(a_s + lds_off(arow + i * 32, chalf));
#pragma unroll
    for (int j = 0; j < 2; ++j) bfr[0][j] = *(const bf16x8*)(b_s + lds_off(brow + j * 32, chalf));
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int c = ks & 1;
      if (ks + 1 < BK / 16) {
        const int cn = (ks + 1) * 2 + chalf;
#pragma unroll
        for (int i = 0; i < 4; ++i) af[c ^ 1][i] = *(const bf16x8*)(a_s + lds_off(arow + i * 32, cn));
#pragma unroll
        for (int j = 0; j < 2; ++j) bfr[c ^ 1][j] = *(const bf16x8*)(b_s + lds_off(brow + j * 32, cn));
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[c][i], bfr[c][j], acc[i][j], 0, 0, 0);
    }
    if (more) ld.store(sA[cur ^ 1], sB[cur ^ 1]);
    __syncthreads();
  }

  epilogue<BM, BN, EPI>(p, acc, m0, n0, wm, wn, lane, c_off);
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
    hipLaunchKernelGGL((gemm_bf16_kernel<256, 128, AK, BKC, EPI>), dim3(tiles, z), dim3(256), 0, s, p);
  } else {
    const int tiles = ((p.M + 255) / 256) * ((p.N + 255) / 256);
    hipLaunchKernelGGL((gemm_bf16_kernel<256, 256, AK, BKC, EPI>), dim3(tiles, z), dim3(512), 0, s, p);
  }
  return hipGetLastError();
}

}  // namespace
