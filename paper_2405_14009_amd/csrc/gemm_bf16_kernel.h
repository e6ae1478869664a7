// bf16 GEMM kernel template on CDNA4 matrix cores: v_mfma_f32_32x32x16_bf16,
// fp32 accumulate.
//
// Tiles.  A BM x BN workgroup tile runs NW waves in a 2 x NW/2 grid; each
// wave owns a 128 x (BN / (NW/2)) tile of 32x32 MFMA blocks.  The launcher
// uses NW = 8: 128 x 64 wave tiles for 256x256 tiles and 128 x 32 for 256x128
// tiles, two waves per SIMD.  With one wave per SIMD (NW = 4, 128 x 128 wave
// tiles) every barrier, LDS-read wait and full memory-instruction queue left
// the matrix core idle; with two, the other wave issues MFMAs meanwhile, which
// measured faster on every stage shape despite the smaller wave tiles.
//
// Staging.  k-tiles of 64 are copied from memory straight into LDS by
// buffer-load-to-LDS instructions (each wave instruction deposits 64 lanes x
// 16 bytes contiguously; out-of-range offsets deposit zeros, so ragged edges
// need no branches and no registers hold tile data).  Two LDS stages: the
// copy of tile t+1 is in flight while tile t is multiplied, one barrier per
// k-tile.
//   * k-contiguous operand: LDS tile [rows][64], 16-byte chunks XOR-swizzled
//     by row; fragments are one ds_read_b128 per lane.
//   * m/n-contiguous operand (the token reduction of the weight-gradient
//     GEMMs, the [in, out] weights in the forward): LDS tile [64][rows] in
//     memory order, chunks XOR-swizzled by k-row; fragments are two
//     ds_read_b64_tr_b16 per lane, which transpose 4x16 blocks across each
//     16-lane group so every lane receives 8 k-consecutive values of its
//     row/column, the same operand layout as the k-contiguous case.
// Within a k-tile the fragments of the next 16-wide k-step are read while the
// current step's MFMAs issue.
#pragma once

#include "gemm.h"
#include "mfma_common.h"

namespace {

constexpr int BK = 64;

// k-contiguous tiles: chunk c (8 elements) of row r lives at chunk c ^ swz_k(r).
// Depends on r mod 32 only (so every 32-row MFMA block of a wave shares it)
// and spreads any 8, and any 16, consecutive rows over distinct banks.
__device__ __forceinline__ int swz_k(int r) { return (r & 7) ^ ((r >> 3) & 3); }
// m/n-contiguous tiles: chunk c of k-row r lives at chunk c ^ swz_mn(r).
__device__ __forceinline__ int swz_mn(int r) { return (r & 3) << 2; }

// One operand's share of the per-k-tile copy: this wave issues instructions
// g = wave + NW q (q < NI) of the operand's 1 KB slices (NW waves).  Every slice of a wave
// differs from its first by a fixed row (k-contiguous) or k-row
// (m/n-contiguous) step, so two per-lane values describe all of them.
template <int ROWS, bool KC, int NI, int NW>
struct Copier {
  uint32_t base;  // byte offset of this lane's row (k-contiguous) / column (m/n-contiguous) in slice 0
  int kk;         // k offset of this lane's data within the k-tile, slice 0
  int mn;         // this lane's row (k-contiguous) / first column (m/n-contiguous), slice 0
  static constexpr int RPI = KC ? 8 : 512 / ROWS;  // rows (k-contiguous) or k-rows per slice
  __device__ __forceinline__ void init(int wave, long ld, int mn0, int lane) {
    if (KC) {
      const int row = 8 * wave + (lane >> 3);
      kk = 8 * ((lane & 7) ^ swz_k(row));  // the same for every slice: rows differ by 32 q
      mn = mn0 + row;
      base = (uint32_t)((long)mn * ld * 2);
    } else {
      constexpr int CPR = ROWS / 8;  // chunks per k-row
      const int krow = RPI * wave + lane / CPR;
      const int c = (lane % CPR) ^ swz_mn(krow);  // k-rows of later slices differ by a multiple of 4
      kk = krow;
      mn = mn0 + 8 * c;
      base = (uint32_t)(2 * mn);
    }
  }
  __device__ __forceinline__ void issue(const i32x4& r, char* tile, int wave, long ld, int MN, int k0,
                                        int K) const {
#pragma unroll
    for (int q = 0; q < NI; ++q) {
      uint32_t off;
      if (KC) {
        const int k = k0 + kk;
        const bool ok = (mn + 8 * NW * q < MN) && (k < K);
        off = ok ? base + (uint32_t)(8 * NW * q) * (uint32_t)(2 * ld) + 2u * k : kOOB;
      } else {
        const int k = k0 + kk + NW * RPI * q;
        off = (mn < MN && k < K) ? base + (uint32_t)k * (uint32_t)(2 * ld) : kOOB;
      }
      dma16(r, __builtin_amdgcn_readfirstlane(lds_addr(tile) + (wave + NW * q) * 1024), off);
    }
  }
};

// Per-lane byte offsets of a wave's MFMA fragments in a staged operand tile.
// k-contiguous: off[ks] for k-step ks (block i of 32 rows adds 4096 i).
// m/n-contiguous: off[b] for 32-row block b (k-step ks adds 32 ks rows of
// the tile, the second half-read 4 k-rows).
template <int ROWS, bool KC, int NBLK>
struct FragOffsets {
  static constexpr int N = KC ? 4 : NBLK;
  uint32_t off[N];
  __device__ __forceinline__ void init(int r0, int lane) {
    if constexpr (KC) {
      const int r = r0 + (lane & 31);
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const int c = ks * 2 + (lane >> 5);
        off[ks] = (uint32_t)(r * 128 + ((c ^ swz_k(r)) << 4));
      }
    } else {
      const int i = lane & 15;
      const int k = 8 * (lane >> 5) + (i >> 2);
#pragma unroll
      for (int b = 0; b < NBLK; ++b) {
        const int mn = r0 + 32 * b + 16 * ((lane >> 4) & 1) + 4 * (i & 3);
        off[b] = (uint32_t)(k * (ROWS * 2) + (((mn >> 3) ^ swz_mn(k)) << 4) + 8 * (i & 1));
      }
    }
  }
};

// Fragment of 32-row block b, k-step ks: 8 k-consecutive values of one row per lane.
template <int ROWS, bool KC, int NBLK>
__device__ __forceinline__ bf16x8 frag(const char* tile, const FragOffsets<ROWS, KC, NBLK>& fo, int b,
                                       int ks) {
  if constexpr (KC) {
    return *(const bf16x8*)(tile + fo.off[ks] + 4096 * b);
  } else {
    const char* p0 = tile + fo.off[b] + 16 * ks * (ROWS * 2);
    const char* p1 = p0 + 4 * (ROWS * 2);  // k + 4 keeps k % 4, hence the swizzle
    s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)p0);
    s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)p1);
    s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8, v);
  }
}

// MFMAs of one staged k-tile for a wave tile of 4 x TN blocks of 32x32.  The
// fragments of k-step ks+1 are read while the MFMAs of k-step ks issue;
// scheduling groups pin that interleave (one MFMA, then that k-step's share
// of LDS reads) so the reads stay ahead of their use.
template <int BM, int BN, bool AK, bool BKC, int TN>
__device__ __forceinline__ void mma_tile(f32x16 (&acc)[4][TN], const char* ta, const char* tb,
                                         const FragOffsets<BM, AK, 4>& fa,
                                         const FragOffsets<BN, BKC, TN>& fb) {
  constexpr int READS = 4 * (AK ? 1 : 2) + TN * (BKC ? 1 : 2);  // LDS read instructions per k-step
  constexpr int NMFMA = 4 * TN;
  constexpr int PER = (READS + NMFMA - 1) / NMFMA;
  bf16x8 af[2][4], bfr[2][TN];
#pragma unroll
  for (int i = 0; i < 4; ++i) af[0][i] = frag(ta, fa, i, 0);
#pragma unroll
  for (int j = 0; j < TN; ++j) bfr[0][j] = frag(tb, fb, j, 0);
  __builtin_amdgcn_sched_group_barrier(0x100, READS, 0);
#pragma unroll
  for (int ks = 0; ks < BK / 16; ++ks) {
    const int c = ks & 1;
    if (ks + 1 < BK / 16) {
#pragma unroll
      for (int i = 0; i < 4; ++i) af[c ^ 1][i] = frag(ta, fa, i, ks + 1);
#pragma unroll
      for (int j = 0; j < TN; ++j) bfr[c ^ 1][j] = frag(tb, fb, j, ks + 1);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[c][i], bfr[c][j], acc[i][j], 0, 0, 0);
    if (ks + 1 < BK / 16) {
#pragma unroll
      for (int q = 0; q < NMFMA; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, PER, 0);
      }
    } else {
      __builtin_amdgcn_sched_group_barrier(0x008, NMFMA, 0);
    }
  }
}

// Epilogue through LDS.  For each 32-row block-row of its tile a wave writes
// its accumulators (MFMA layout: lane l holds column l % 32, rows
// 8 (r / 4) + 4 (l / 32) + r % 4) to a row-major fp32 LDS tile (rows padded by
// 8 floats so the two half-waves hit disjoint banks), then re-reads it row by
// row so each lane applies the epilogue to 4 consecutive columns with vector
// global accesses.  `sm` is this wave's private LDS region.
template <int EPI, int TN>
__device__ __forceinline__ void epilogue(const GemmParams& p, f32x16 (&acc)[4][TN], float* sm, int m0,
                                         int n0, int lane, long c_off) {
  constexpr int COLS = 32 * TN, STRIDE = COLS + 8;
  typedef typename EpiOut<EPI, bf16>::type OutT;
  void* C = (OutT*)p.C + c_off;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        sm[(8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * STRIDE + 32 * j + (lane & 31)] = acc[i][j][r];
    __builtin_amdgcn_wave_barrier();
#pragma unroll 2
    for (int q = 0; q < COLS / 8; ++q) {
      const int idx = lane + 64 * q;
      const int row = idx / (COLS / 4), c4 = idx % (COLS / 4);
      const float4 v = *(const float4*)(sm + row * STRIDE + 4 * c4);
      const int m = m0 + i * 32 + row, n = n0 + 4 * c4;
      if (m < p.M && n < p.N) epi_store4<EPI, bf16>(p, C, m, n, v);
    }
    __builtin_amdgcn_wave_barrier();
  }
}

template <int BM, int BN, int NW, bool AK, bool BKC, int EPI>
__global__ __launch_bounds__(64 * NW) void gemm_bf16_kernel(GemmParams p) {
  static_assert(BM == 256 && (BN == 256 || BN == 128) && (NW == 4 || NW == 8), "tile shapes");
  constexpr int WN_ = NW / 2;            // waves along n (2 along m)
  constexpr int TN = BN / (32 * WN_);    // 32-wide blocks per wave along n
  constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2;
  constexpr int STAGE = A_BYTES + B_BYTES;
  constexpr int NA = A_BYTES / 1024, NB = B_BYTES / 1024;  // wave instructions per k-tile
  static_assert(NA % NW == 0 && NB % NW == 0, "copy split");
  constexpr int NIA = NA / NW, NIB = NB / NW;
  // Two stages as distinct LDS objects, so the compiler can tell that the
  // copy into one stage does not alias the fragment reads from the other.
  __shared__ __attribute__((aligned(1024))) char lds0[STAGE];
  __shared__ __attribute__((aligned(1024))) char lds1[STAGE];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
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
  const i32x4 ra = make_rsrc(A, 2L * (AK ? (long)p.M * p.lda : (long)p.K * p.lda));
  const i32x4 rb = make_rsrc(B, 2L * (BKC ? (long)p.N * p.ldb : (long)p.K * p.ldb));

  int kb = 0, ke = p.K;
  if (p.krange == KR_BELOW) ke = min(p.K, m0 + BM);
  else if (p.krange == KR_ABOVE) kb = (m0 / BK) * BK;
  const int nk = ke > kb ? (ke - kb + BK - 1) / BK : 0;

  Copier<BM, AK, NIA, NW> ca;
  Copier<BN, BKC, NIB, NW> cb;
  ca.init(wave, p.lda, m0, lane);
  cb.init(wave, p.ldb, n0, lane);
  FragOffsets<BM, AK, 4> fa;
  FragOffsets<BN, BKC, TN> fb;
  fa.init(wm * 128, lane);
  fb.init(wn * (BN / WN_), lane);

  f32x16 acc[4][TN];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // Tile t lives in stage t % 2.  The copy of tile t+1 is issued before the
  // MFMAs of tile t.  With a segmented reduction the k-tile's segment selects
  // the operand bases (a k-tile never straddles segments).
  auto issue = [&](char* st, int k0) {
    if (p.kseg_len > 0) {
      const int sg = k0 / p.kseg_len, kin = k0 - sg * p.kseg_len;
      const i32x4 sa = make_rsrc((const bf16*)p.segA[sg] + zb * p.a_bs + zh * p.a_hs,
                                 2L * (AK ? (long)p.M * p.lda : (long)p.kseg_len * p.lda));
      const i32x4 sb = make_rsrc((const bf16*)p.segB[sg] + zb * p.b_bs + zh * p.b_hs,
                                 2L * (BKC ? (long)p.N * p.ldb : (long)p.kseg_len * p.ldb));
      ca.issue(sa, st, wave, p.lda, p.M, kin, p.kseg_len);
      cb.issue(sb, st + A_BYTES, wave, p.ldb, p.N, kin, p.kseg_len);
    } else {
      ca.issue(ra, st, wave, p.lda, p.M, k0, ke);
      cb.issue(rb, st + A_BYTES, wave, p.ldb, p.N, k0, ke);
    }
  };
  if (nk > 0) issue(lds0, kb);
  stage_sync();
  int t = 0;
  for (; t + 1 < nk; t += 2) {
    issue(lds1, kb + (t + 1) * BK);
    mma_tile<BM, BN, AK, BKC, TN>(acc, lds0, lds0 + A_BYTES, fa, fb);
    stage_sync();
    if (t + 2 < nk) issue(lds0, kb + (t + 2) * BK);
    mma_tile<BM, BN, AK, BKC, TN>(acc, lds1, lds1 + A_BYTES, fa, fb);
    stage_sync();
  }
  if (t < nk) mma_tile<BM, BN, AK, BKC, TN>(acc, lds0, lds0 + A_BYTES, fa, fb);

  // LDS is free once every wave is past its last k-tile.
  __syncthreads();
  constexpr int EPI_BYTES = 32 * (32 * TN + 8) * 4;  // one wave's block-row tile
  static_assert((NW / 2) * EPI_BYTES <= STAGE, "epilogue tiles fit NW/2 per stage");
  float* sm = (float*)((wave < NW / 2 ? lds0 : lds1) + (wave % (NW / 2)) * EPI_BYTES);
  epilogue<EPI, TN>(p, acc, sm, m0 + wm * 128, n0 + wn * (BN / WN_), lane, c_off);
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
  // 8 waves (2 per SIMD): while one wave of a SIMD waits on a barrier or
  // its LDS reads, the other issues MFMAs.
  if (p.N <= 128 || cost(256, 128) < cost(256, 256)) {
    const int tiles = ((p.M + 255) / 256) * ((p.N + 127) / 128);
    hipLaunchKernelGGL((gemm_bf16_kernel<256, 128, 8, AK, BKC, EPI>), dim3(tiles, z), dim3(512), 0, s, p);
  } else {
    const int tiles = ((p.M + 255) / 256) * ((p.N + 255) / 256);
    hipLaunchKernelGGL((gemm_bf16_kernel<256, 256, 8, AK, BKC, EPI>), dim3(tiles, z), dim3(512), 0, s, p);
  }
  return hipGetLastError();
}

}  // namespace
