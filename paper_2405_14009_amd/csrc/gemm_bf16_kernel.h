// bf16 GEMM kernels on CDNA4 matrix cores: v_mfma_f32_32x32x16_bf16,
// fp32 accumulate.  Two kernels share the staging and fragment machinery:
//   gemm_bf16_kernel     256 x 256 workgroup tiles;
//   gemm_bf16_pp_kernel  256 x 128 tiles with a ping-pong schedule and a
//                        k-split into two wave groups.
//
// Tiles.  A BM x BN workgroup tile runs NW = 8 waves in KS k-groups; each
// k-group is a 2 x (NW / KS / 2) grid of 128 x (BN / (NW / KS / 2)) wave tiles
// of 32x32 MFMA blocks covering the whole workgroup tile.  With eight waves
// every SIMD runs two, so while one waits on a barrier or on its LDS reads the
// other issues MFMAs (one wave per SIMD with 128 x 128 wave tiles left the
// matrix core idle at every such wait).
//
// Staging.  k-tiles of BK are copied from memory straight into LDS by
// buffer-load-to-LDS instructions (each wave instruction deposits 64 lanes x
// 16 bytes contiguously; out-of-range offsets deposit zeros, so ragged edges
// need no branches and no registers hold tile data).  NST stages form a ring:
// the copy of tile t + NST - 1 is issued while tile t is multiplied, its A
// and B slices at separate points of the first k-steps; a wave waits only for
// its own copies of the oldest stage (vmcnt of the copies issued after it),
// then one barrier per k-tile publishes that stage and frees the one
// multiplied before.
//   * k-contiguous operand: LDS tile [rows][BK], 16-byte chunks XOR-swizzled
//     by row; fragments are one ds_read_b128 per lane.
//   * m/n-contiguous operand (the token reduction of the weight-gradient
//     GEMMs, the [in, out] weights in the forward): LDS tile [BK][rows] in
//     memory order, chunks XOR-swizzled by k-row; fragments are two
//     ds_read_b64_tr_b16 per lane, which transpose 4x16 blocks across each
//     16-lane group so every lane receives 8 k-consecutive values of its
//     row/column, the same operand layout as the k-contiguous case.
//
// What bounds these kernels on MI355X (counters, and variants with one
// component switched off): the copies.  A CU keeps 60-85 L2 read requests of
// 128 bytes in flight at 350-450 cycles of average latency, so it receives
// 20-25 bytes per clock, while a 256 x 256 x 64 k-tile (64 KB) feeds 2048 MFMA
// cycles per SIMD (32 bytes per clock at the full rate); the units that return
// the copied lines to LDS are busy about 70 % of the time.  Without the copies
// the same kernels reach 1.5-1.9 PFLOP/s; without the fragment reads they
// barely change.  Where in the multiply of a k-tile the next refill is issued
// matters (5-12 %, see the kernels); deeper rings of 32-deep k-tiles, register
// staging (buffer_load + ds_write, also two k-tiles ahead), an L2 prefetch of
// the k-tile after next, padded leading dimensions and a one-wave-per-SIMD
// layout did not help; the ping-pong schedule and a tile
// order whose 32 concurrent tiles per XCD share fewer operand panels did
// (256 x 128 tiles).
#pragma once

#include <algorithm>

#include "gemm.h"
#include "mfma_common.h"

namespace {

// k-contiguous tiles (64-deep k-tiles, 8 chunks of 16 bytes per row): chunk
// c (8 elements) of row r lives at chunk c ^ swz_k<BK>(r).  Depends on r mod
// 32 only (so every 32-row MFMA block of a wave shares it) and places the 16
// rows that one ds_read_b128 pass serves (16 lanes x 16 bytes, two rows per
// 256-byte window) on distinct 16-byte bank groups.
template <int BK>
__device__ __forceinline__ int swz_k(int r) {
  static_assert(BK == 64, "k-tiles of 64");
  return (r & 7) ^ ((r >> 3) & 3);
}
// m/n-contiguous tiles: chunk c of k-row r lives at chunk c ^ swz_mn(r).
__device__ __forceinline__ int swz_mn(int r) { return (r & 3) << 2; }

// One operand's share of the per-k-tile copy: this wave issues instructions
// g = wave + NW q (q < NI) of the operand's 1 KB slices (NW waves).  Every slice of a wave
// differs from its first by a fixed row (k-contiguous) or k-row
// (m/n-contiguous) step, so two per-lane values describe all of them.
template <int ROWS, bool KC, int NI, int NW, int BK>
struct Copier {
  uint32_t base;  // byte offset of this lane's row (k-contiguous) / column (m/n-contiguous) in slice 0
  int kk;         // k offset of this lane's data within the k-tile, slice 0
  int mn;         // this lane's row (k-contiguous) / first column (m/n-contiguous), slice 0
  static constexpr int CPR = KC ? BK / 8 : ROWS / 8;  // 16-byte chunks per LDS row
  static constexpr int RPI = 64 / CPR;                 // LDS rows (k-rows if m/n-contiguous) per slice
  static_assert(KC || (NW * RPI) % 4 == 0, "slices of a wave keep k mod 4, hence the swizzle");
  __device__ __forceinline__ void init(int wave, long ld, int mn0, int lane) {
    if (KC) {
      const int row = RPI * wave + lane / CPR;
      kk = 8 * ((lane % CPR) ^ swz_k<BK>(row));  // the same for every slice: rows differ by 64 q
      mn = mn0 + row;
      base = (uint32_t)((long)mn * ld * 2);
    } else {
      const int krow = RPI * wave + lane / CPR;
      const int c = (lane % CPR) ^ swz_mn(krow);
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
        const bool ok = (mn + RPI * NW * q < MN) && (k < K);
        off = ok ? base + (uint32_t)(RPI * NW * q) * (uint32_t)(2 * ld) + 2u * k : kOOB;
      } else {
        const int k = k0 + kk + NW * RPI * q;
        off = (mn < MN && k < K) ? base + (uint32_t)k * (uint32_t)(2 * ld) : kOOB;
      }
      dma16(r, __builtin_amdgcn_readfirstlane(lds_addr(tile) + (wave + NW * q) * 1024), off);
    }
  }
};

// Column sums over k of the staged m/n-contiguous B tiles ([BK][BN] bf16,
// 16-byte chunks swizzled by k-row), accumulated over the k-tiles a
// workgroup takes part for: thread t (of 512) owns chunk column t % (BN / 8)
// and k-rows t / (BN / 8) + R i of every tile (R row groups), 8 fp32 partial
// sums.  finish() adds the R partials of each column in a fixed order through
// LDS and stores the workgroup's row of partial sums, so the result is
// reproducible.
template <int BN, int BK>
struct ColSums {
  static constexpr int CC = BN / 8, R = 512 / CC, RPT = BK / R;
  static_assert(BK % R == 0, "row groups");
  static constexpr int RED_BYTES = R * BN * 4;
  float s[8];
  int cc, rg;
  __device__ __forceinline__ void init(int tid) {
    cc = tid % CC;
    rg = tid / CC;
#pragma unroll
    for (int e = 0; e < 8; ++e) s[e] = 0.f;
  }
  __device__ __forceinline__ void tile(const char* tb) {
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const int k = rg + R * i;
      const uint4 v = *(const uint4*)(tb + k * (BN * 2) + ((cc ^ swz_mn(k)) << 4));
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        s[2 * e] += __uint_as_float(w[e] << 16);
        s[2 * e + 1] += __uint_as_float(w[e] & 0xffff0000u);
      }
    }
  }
  // red: RED_BYTES of LDS that no wave touches meanwhile; every wave calls it.
  __device__ __forceinline__ void finish(float* red, const GemmParams& p, int tm, int n0, int tid) {
#pragma unroll
    for (int e = 0; e < 8; ++e) red[rg * BN + 8 * cc + e] = s[e];
    __syncthreads();
    if (tid < BN) {
      float t = 0.f;
#pragma unroll 8
      for (int r = 0; r < R; ++r) t += red[r * BN + tid];
      const int n = n0 + tid;
      if (n < p.N) p.colsum_work[(long)tm * p.N + n] = t;
    }
    __syncthreads();
  }
};

// Per-lane byte offsets of a wave's MFMA fragments in a staged operand tile.
// k-contiguous: off[ks] for k-step ks (block i of 32 rows adds 64 BK i).
// m/n-contiguous: off[b] for 32-row block b (k-step ks adds 16 ks rows of
// the tile, the second half-read 4 k-rows).
template <int ROWS, bool KC, int NBLK, int NKS, int BK>
struct FragOffsets {
  static constexpr int N = KC ? NKS : NBLK;
  uint32_t off[N];
  // ks0: the first of the NKS k-steps of the k-tile that this wave multiplies.
  __device__ __forceinline__ void init(int r0, int lane, int ks0) {
    if constexpr (KC) {
      const int r = r0 + (lane & 31);
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const int c = (ks0 + ks) * 2 + (lane >> 5);
        off[ks] = (uint32_t)(r * (2 * BK) + ((c ^ swz_k<BK>(r)) << 4));
      }
    } else {
      const int i = lane & 15;
      const int k = 16 * ks0 + 8 * (lane >> 5) + (i >> 2);
#pragma unroll
      for (int b = 0; b < NBLK; ++b) {
        const int mn = r0 + 32 * b + 16 * ((lane >> 4) & 1) + 4 * (i & 3);
        off[b] = (uint32_t)(k * (ROWS * 2) + (((mn >> 3) ^ swz_mn(k)) << 4) + 8 * (i & 1));
      }
    }
  }
};

// Fragment of 32-row block b, k-step ks: 8 k-consecutive values of one row per lane.
template <int ROWS, bool KC, int NBLK, int NKS, int BK>
__device__ __forceinline__ bf16x8 frag(const char* tile, const FragOffsets<ROWS, KC, NBLK, NKS, BK>& fo,
                                       int b, int ks) {
  if constexpr (KC) {
    return *(const bf16x8*)(tile + fo.off[ks] + 64 * BK * b);
  } else {
    const char* p0 = tile + fo.off[b] + 16 * ks * (ROWS * 2);
    const char* p1 = p0 + 4 * (ROWS * 2);  // k + 4 keeps k % 4, hence the swizzle
    s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)p0);
    s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)p1);
    s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8, v);
  }
}

// MFMAs of one staged k-tile for a wave tile of 4 x TN blocks of 32x32 over
// NKS k-steps.  The fragments of k-step ks+1 are read while the MFMAs of
// k-step ks issue; scheduling groups pin that interleave (one MFMA, then that
// k-step's share of LDS reads) so the reads stay ahead of their use.
// step(ks) runs at the head of k-step ks, after the fragment reads issued
// before it (the kernels issue their next k-tile's copies from it).
// DEFER: the MFMAs of the last k-step are left for the next call, which
// issues them from (pa, pb) right behind its first fragment reads, so the
// matrix core has work while those reads are in flight after the k-tile
// barrier; mma_flush adds the last pending product.  (Zero fragments make the
// first call's pending MFMAs a no-op.)
template <int TN>
__device__ __forceinline__ void mma_flush(f32x16 (&acc)[4][TN], const bf16x8 (&pa)[4], const bf16x8 (&pb)[TN]) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pa[i], pb[j], acc[i][j], 0, 0, 0);
}
template <int TN>
__device__ __forceinline__ void mma_pending_clear(bf16x8 (&pa)[4], bf16x8 (&pb)[TN]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) pa[i] = bf16x8{};
#pragma unroll
  for (int j = 0; j < TN; ++j) pb[j] = bf16x8{};
}
template <int BM, int BN, bool AK, bool BKC, int TN, int NKS, int BK, bool DEFER, typename Step>
__device__ __forceinline__ void mma_tile(f32x16 (&acc)[4][TN], const char* ta, const char* tb,
                                         const FragOffsets<BM, AK, 4, NKS, BK>& fa,
                                         const FragOffsets<BN, BKC, TN, NKS, BK>& fb, Step step,
                                         bf16x8 (&pa)[4], bf16x8 (&pb)[TN]) {
  constexpr int READS = 4 * (AK ? 1 : 2) + TN * (BKC ? 1 : 2);  // LDS read instructions per k-step
  constexpr int NMFMA = 4 * TN;
  constexpr int PER = (READS + NMFMA - 1) / NMFMA;
  bf16x8 af[2][4], bfr[2][TN];
#pragma unroll
  for (int i = 0; i < 4; ++i) af[0][i] = frag(ta, fa, i, 0);
#pragma unroll
  for (int j = 0; j < TN; ++j) bfr[0][j] = frag(tb, fb, j, 0);
  __builtin_amdgcn_sched_group_barrier(0x100, READS, 0);
  if constexpr (DEFER) {
    mma_flush<TN>(acc, pa, pb);
    __builtin_amdgcn_sched_group_barrier(0x008, NMFMA, 0);
  }
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    const int c = ks & 1;
    __builtin_amdgcn_sched_barrier(0);
    step(ks);
    __builtin_amdgcn_sched_barrier(0);
    if (ks + 1 < NKS) {
#pragma unroll
      for (int i = 0; i < 4; ++i) af[c ^ 1][i] = frag(ta, fa, i, ks + 1);
#pragma unroll
      for (int j = 0; j < TN; ++j) bfr[c ^ 1][j] = frag(tb, fb, j, ks + 1);
    }
    if (DEFER && ks + 1 == NKS) {
#pragma unroll
      for (int i = 0; i < 4; ++i) pa[i] = af[c][i];
#pragma unroll
      for (int j = 0; j < TN; ++j) pb[j] = bfr[c][j];
      break;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[c][i], bfr[c][j], acc[i][j], 0, 0, 0);
    if (ks + 1 < NKS) {
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

// Epilogue through LDS.  For each 32-row block-row i in [I0, I1) of its tile
// a wave writes its accumulators (MFMA layout: lane l holds column l % 32,
// rows 8 (r / 4) + 4 (l / 32) + r % 4) to a row-major fp32 LDS tile (rows
// padded by 8 floats so the two half-waves hit disjoint banks), then re-reads
// it row by row so each lane applies the epilogue to 4 consecutive columns
// with vector global accesses.  `sm` is this wave's private LDS region.
// Epilogues with a per-element input (residual, GeLU input, gradient being
// accumulated) fetch the next block-row's inputs while the current one is
// finished, so those loads overlap instead of each costing a round trip
// (LOOK; without it each block-row's inputs are fetched as it is finished,
// which needs 32 fewer registers).
template <int EPI, int TN, int I0, int I1, bool LOOK = true>
__device__ __forceinline__ void epilogue(const GemmParams& p, f32x16 (&acc)[4][TN], float* sm, int m0,
                                         int n0, int lane, long c_off) {
  constexpr int COLS = 32 * TN, STRIDE = COLS + 8;
  constexpr int NQ = COLS / 8;  // 4-column groups per lane per block-row
  constexpr bool IN = EpiIn<EPI>::kHas;
  typedef typename EpiOut<EPI, bf16>::type OutT;
  void* C = (OutT*)p.C + c_off;
  static_assert(64 % (COLS / 4) == 0, "a lane keeps its columns on every row");
  float4 bias = make_float4(0.f, 0.f, 0.f, 0.f);
  if constexpr (epi_has_bias(EPI)) {
    const int n = n0 + 4 * (lane % (COLS / 4));
    if (n < p.N) bias = *(const float4*)(p.bias + n);
  }
  EpiIn<EPI> in[2][NQ];
  auto fetch = [&](int i, EpiIn<EPI>(&dst)[NQ]) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int idx = lane + 64 * q;
      const int m = m0 + i * 32 + idx / (COLS / 4), n = n0 + 4 * (idx % (COLS / 4));
      if (m < p.M && n < p.N) dst[q] = epi_fetch4<EPI, bf16>(p, C, m, n);
    }
  };
  if constexpr (IN && LOOK) fetch(I0, in[0]);
#pragma unroll
  for (int i = I0; i < I1; ++i) {
    const int cur = (i - I0) & 1;
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        sm[(8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * STRIDE + 32 * j + (lane & 31)] = acc[i][j][r];
    __builtin_amdgcn_wave_barrier();
    // The next block-row's inputs are requested once this row's accumulators
    // are in LDS (their registers are free by then).
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (IN && LOOK) {
      if (i + 1 < I1) fetch(i + 1, in[cur ^ 1]);
    }
    if constexpr (IN && !LOOK) fetch(i, in[cur]);
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int idx = lane + 64 * q;
      const int row = idx / (COLS / 4), c4 = idx % (COLS / 4);
      const float4 v = *(const float4*)(sm + row * STRIDE + 4 * c4);
      const int m = m0 + i * 32 + row, n = n0 + 4 * c4;
      if (m < p.M && n < p.N) epi_finish4<EPI, bf16>(p, C, m, n, v, in[cur][q], bias);
    }
    __builtin_amdgcn_wave_barrier();
  }
}

// Reduction of a k-split workgroup: the two k-groups hold partial sums of the
// same output tile.  Wave (g, w) hands the partial of the block-rows that the
// other group finishes (rows 2 (1 - g), +1) to its partner through LDS slot
// `mine`, then adds the partner's partial of its own rows (2 g, +1) from slot
// `theirs`.  Slots hold [row-block][n-block][register][lane] floats, so every
// access is 256 contiguous bytes per wave instruction.
template <int TN, int G>
__device__ __forceinline__ void ksplit_reduce(f32x16 (&acc)[4][TN], float* mine, const float* theirs,
                                              int lane) {
#pragma unroll
  for (int il = 0; il < 2; ++il)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) mine[((il * TN + j) * 16 + r) * 64 + lane] = acc[2 * (1 - G) + il][j][r];
  __syncthreads();
#pragma unroll
  for (int il = 0; il < 2; ++il)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[2 * G + il][j][r] += theirs[((il * TN + j) * 16 + r) * 64 + lane];
}

// s_waitcnt vmcnt(N), other counters untouched (gfx9 encoding: vmcnt bits
// [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8]).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}

template <int BM, int BN, int NW, int KS, int BK, int NST, bool AK, bool BKC, int EPI>
__global__ __launch_bounds__(64 * NW) void gemm_bf16_kernel(GemmParams p) {
  // the configuration the launcher uses (256 x 128 tiles run the ping-pong
  // kernel, which owns the k-split)
  static_assert(BM == 256 && BN == 256 && NW == 8 && KS == 1 && BK == 64 && NST >= 2, "tile shapes");
  constexpr int NWS = NW / KS;           // waves per k-group
  constexpr int WN_ = NWS / 2;           // waves along n (2 along m)
  constexpr int TN = BN / (32 * WN_);    // 32-wide blocks per wave along n
  constexpr int NKS = (BK / 16) / KS;    // k-steps per wave per k-tile
  constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2;
  constexpr int STAGE = A_BYTES + B_BYTES;
  constexpr int NA = A_BYTES / 1024, NB = B_BYTES / 1024;  // wave instructions per k-tile
  static_assert(NA % NW == 0 && NB % NW == 0, "copy split");
  constexpr int NIA = NA / NW, NIB = NB / NW;
  constexpr int PER_TILE = NIA + NIB;    // copy instructions per wave per k-tile
  constexpr int EPI_BYTES = 32 * (32 * TN + 8) * 4;  // one wave's epilogue block-row tile
  constexpr int LDS_BYTES = NST * STAGE > NW * EPI_BYTES ? NST * STAGE : NW * EPI_BYTES;
  static_assert(LDS_BYTES <= 160 * 1024, "LDS");
  __shared__ __attribute__((aligned(1024))) char lds[LDS_BYTES];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int kg = wave / NWS, ws = wave % NWS;
  const int wm = ws / WN_, wn = ws % WN_;

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

  Copier<BM, AK, NIA, NW, BK> ca;
  Copier<BN, BKC, NIB, NW, BK> cb;
  ca.init(wave, p.lda, m0, lane);
  cb.init(wave, p.ldb, n0, lane);
  FragOffsets<BM, AK, 4, NKS, BK> fa;
  FragOffsets<BN, BKC, TN, NKS, BK> fb;
  fa.init(wm * 128, lane, kg * NKS);
  fb.init(wn * (BN / WN_), lane, kg * NKS);

  f32x16 acc[4][TN];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  // column sums of B (a workgroup-uniform condition)
  constexpr bool CS = !AK && !BKC;  // weight-gradient layout only
  // Every tile-row takes part in the column sums for one k-tile in tiles_m, so
  // the extra work spreads evenly over the launch.
  const bool cs_on = CS && p.colsum_out != nullptr && z == 0;
  int cs_next = tm;  // next k-tile this workgroup sums
  ColSums<BN, BK> cs;
  if (cs_on) cs.init(threadIdx.x);

  // Operands of the k-tile at k0: with a segmented reduction the k-tile's
  // segment selects the operand bases (a k-tile never straddles segments).
  struct Src {
    i32x4 a, b;
    int k, kend;
  };
  auto source = [&](int k0) {
    Src r{ra, rb, k0, ke};
    if (p.kseg_len > 0) {
      const int sg = k0 / p.kseg_len;
      r.k = k0 - sg * p.kseg_len;
      r.kend = p.kseg_len;
      r.a = make_rsrc((const bf16*)p.segA[sg] + zb * p.a_bs + zh * p.a_hs,
                      2L * (AK ? (long)p.M * p.lda : (long)p.kseg_len * p.lda));
      r.b = make_rsrc((const bf16*)p.segB[sg] + zb * p.b_bs + zh * p.b_hs,
                      2L * (BKC ? (long)p.N * p.ldb : (long)p.kseg_len * p.ldb));
    }
    return r;
  };
  auto issue = [&](char* st, int k0) {
    const Src sr = source(k0);
    ca.issue(sr.a, st, wave, p.lda, p.M, sr.k, sr.kend);
    cb.issue(sr.b, st + A_BYTES, wave, p.ldb, p.N, sr.k, sr.kend);
  };
  // Ring of NST stages: tile t lives in stage t mod NST.  Tiles 0 .. NST-2 are
  // issued up front; iteration t waits for tile t, publishes it with the
  // barrier (which also certifies that every wave is done with tile t-1), then
  // refills tile t-1's stage with tile t + NST - 1 while it multiplies tile t:
  // the A slices at the head of the first k-step, the B slices at the head of
  // the second (one burst of all of them ahead of the first MFMAs held those
  // MFMAs back: 5-11 % longer products).
  // The weight-gradient layout defers each k-tile's last MFMAs (mma_tile):
  // 1-4 % shorter products there; the other layouts measured slower with it.
  static_assert(NKS >= 2, "the refill spans two k-steps");
  constexpr bool DEFER = !AK && !BKC;
  bf16x8 pa[4], pb[TN];
  mma_pending_clear<TN>(pa, pb);
#pragma unroll
  for (int i = 0; i < NST - 1; ++i)
    if (i < nk) issue(lds + i * STAGE, kb + i * BK);
  int sc = 0, si = NST - 1;  // stage of tile t, stage that tile t + NST - 1 goes to
  for (int t = 0; t < nk; ++t) {
    __builtin_amdgcn_sched_barrier(0);
    if (t + NST - 2 < nk) wait_vmcnt<(NST - 2) * PER_TILE>();  // tiles t+1 .. t+NST-2 may stay in flight
    else wait_vmcnt<0>();
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
    const bool refill = t + NST - 1 < nk;
    const Src nx = source(refill ? kb + (t + NST - 1) * BK : kb);
    char* dst = lds + si * STAGE;
    const char* st = lds + sc * STAGE;
    mma_tile<BM, BN, AK, BKC, TN, NKS, BK, DEFER>(acc, st, st + A_BYTES, fa, fb, [&](int ks) {
      if (refill && ks == 0) ca.issue(nx.a, dst, wave, p.lda, p.M, nx.k, nx.kend);
      if (refill && ks == 1) cb.issue(nx.b, dst + A_BYTES, wave, p.ldb, p.N, nx.k, nx.kend);
    }, pa, pb);
    if constexpr (CS) {
      // while the tile's MFMAs drain; the stage stays valid until the next barrier
      __builtin_amdgcn_sched_barrier(0);
      if (cs_on && t == cs_next) {
        cs.tile(st + A_BYTES);
        cs_next += tiles_m;
      }
    }
    sc = sc + 1 == NST ? 0 : sc + 1;
    si = si + 1 == NST ? 0 : si + 1;
  }

  if constexpr (DEFER) mma_flush<TN>(acc, pa, pb);
  // LDS is free once every wave is past its last k-tile.
  __builtin_amdgcn_sched_barrier(0);
  __syncthreads();
  static_assert(ColSums<BN, BK>::RED_BYTES <= LDS_BYTES, "column-sum reduction fits LDS");
  if constexpr (CS) {
    if (cs_on) cs.finish((float*)lds, p, tm, n0, threadIdx.x);
  }
  float* sm = (float*)(lds + wave * EPI_BYTES);
  epilogue<EPI, TN, 0, 4>(p, acc, sm, m0 + wm * 128, n0 + wn * (BN / WN_), lane, c_off);
}

// Persistent form of gemm_bf16_kernel (256 x 256 tiles, 8 waves, two-stage
// ring) for launches of more than one round of tiles.  The grid holds one
// workgroup per compute unit; workgroup q of XCD x (blockIdx.x = x + 8 q)
// walks the tiles x * ntiles / 8 + q, + nq, + 2 nq, ... of the same tile order
// as the one-tile-per-workgroup kernel, so the tiles one XCD runs at a time
// are the ones that share operand panels in its L2.  Between two tiles the
// next tile's first k-tile is copied into stage 0 before the finished tile's
// epilogue runs, and the epilogue stages its rows through LDS above stage 0,
// so that copy is in flight while the epilogue computes and stores.  DEFER:
// each k-tile's last MFMAs are deferred as mma_tile describes.
// Requirements (checked by the launcher): batch * heads == 1, ntiles % 8 == 0.
template <int EPI, bool AK, bool BKC, bool DEFER>
__global__ __launch_bounds__(512) void gemm_bf16_persist_kernel(GemmParams p) {
  constexpr int BM = 256, BN = 256, NW = 8, BK = 64, NST = 2;
  constexpr int WN_ = 4, TN = 2, NKS = 4;
  constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2;
  constexpr int STAGE = A_BYTES + B_BYTES;
  constexpr int NIA = A_BYTES / 1024 / NW, NIB = B_BYTES / 1024 / NW;
  constexpr int EPI_BYTES = 32 * (32 * TN + 8) * 4;
  constexpr int LDS_BYTES = NST * STAGE > STAGE + NW * EPI_BYTES ? NST * STAGE : STAGE + NW * EPI_BYTES;
  static_assert(LDS_BYTES <= 160 * 1024, "LDS");
  static_assert(ColSums<BN, BK>::RED_BYTES <= NW * EPI_BYTES, "column-sum reduction fits above stage 0");
  __shared__ __attribute__((aligned(1024))) char lds[LDS_BYTES];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / WN_, wn = wave % WN_;
  const int tiles_m = (p.M + BM - 1) / BM, tiles_n = (p.N + BN - 1) / BN;
  const int nx = tiles_m * tiles_n / 8;             // tiles of one XCD
  const int xcd = blockIdx.x & 7, nq = gridDim.x >> 3;
  constexpr int GM = 8;
  const int width = GM * tiles_n;
  auto tile_of = [&](int i, int& m0, int& n0, int& tm) {
    const int pid = xcd * nx + i;
    const int first_m = (pid / width) * GM;
    const int gsz = min(tiles_m - first_m, GM);
    tm = first_m + (pid % width) % gsz;
    m0 = tm * BM;
    n0 = ((pid % width) / gsz) * BN;
  };

  const bf16* A = (const bf16*)p.A;
  const bf16* B = (const bf16*)p.B;
  const i32x4 ra = make_rsrc(A, 2L * (AK ? (long)p.M * p.lda : (long)p.K * p.lda));
  const i32x4 rb = make_rsrc(B, 2L * (BKC ? (long)p.N * p.ldb : (long)p.K * p.ldb));
  const int nk = (p.K + BK - 1) / BK;

  Copier<BM, AK, NIA, NW, BK> ca;
  Copier<BN, BKC, NIB, NW, BK> cb;
  FragOffsets<BM, AK, 4, NKS, BK> fa;
  FragOffsets<BN, BKC, TN, NKS, BK> fb;
  fa.init(wm * 128, lane, 0);
  fb.init(wn * (BN / WN_), lane, 0);
  struct Src {
    i32x4 a, b;
    int k, kend;
  };
  auto source = [&](int k0) {
    Src r{ra, rb, k0, p.K};
    if (p.kseg_len > 0) {
      const int sg = k0 / p.kseg_len;
      r.k = k0 - sg * p.kseg_len;
      r.kend = p.kseg_len;
      r.a = make_rsrc(p.segA[sg], 2L * (AK ? (long)p.M * p.lda : (long)p.kseg_len * p.lda));
      r.b = make_rsrc(p.segB[sg], 2L * (BKC ? (long)p.N * p.ldb : (long)p.kseg_len * p.ldb));
    }
    return r;
  };
  auto issue = [&](char* st, int k0) {
    const Src sr = source(k0);
    ca.issue(sr.a, st, wave, p.lda, p.M, sr.k, sr.kend);
    cb.issue(sr.b, st + A_BYTES, wave, p.ldb, p.N, sr.k, sr.kend);
  };
  constexpr bool CS = !AK && !BKC;
  const bool cs_on = CS && p.colsum_out != nullptr;

  int i = blockIdx.x >> 3;
  if (i >= nx) return;
  int m0, n0, tm;
  tile_of(i, m0, n0, tm);
  ca.init(wave, p.lda, m0, lane);
  cb.init(wave, p.ldb, n0, lane);
  if (nk > 0) issue(lds, 0);
  f32x16 acc[4][TN];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][j][r] = 0.f;
  while (true) {
    int cs_next = tm;
    ColSums<BN, BK> cs;
    if (cs_on) cs.init(threadIdx.x);
    int sc = 0, si = 1;
    bf16x8 pa[4], pb[TN];  // the deferred last k-step of each k-tile (mma_tile)
    mma_pending_clear<TN>(pa, pb);
    for (int t = 0; t < nk; ++t) {
      __builtin_amdgcn_sched_barrier(0);
      wait_vmcnt<0>();
      __syncthreads();
      __builtin_amdgcn_sched_barrier(0);
      // refill split over the first two k-steps as in gemm_bf16_kernel
      const bool refill = t + 1 < nk;
      const Src nx = source(refill ? (t + 1) * BK : 0);
      char* dst = lds + si * STAGE;
      const char* st = lds + sc * STAGE;
      mma_tile<BM, BN, AK, BKC, TN, NKS, BK, DEFER>(acc, st, st + A_BYTES, fa, fb, [&](int ks) {
        if (refill && ks == 0) ca.issue(nx.a, dst, wave, p.lda, p.M, nx.k, nx.kend);
        if (refill && ks == 1) cb.issue(nx.b, dst + A_BYTES, wave, p.ldb, p.N, nx.k, nx.kend);
      }, pa, pb);
      if constexpr (CS) {
        __builtin_amdgcn_sched_barrier(0);
        if (cs_on && t == cs_next) {
          cs.tile(st + A_BYTES);
          cs_next += tiles_m;
        }
      }
      sc ^= 1;
      si ^= 1;
    }
    if constexpr (DEFER) mma_flush<TN>(acc, pa, pb);
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();  // every wave is past the last k-tile: both stages are free
    const int cm0 = m0, cn0 = n0, ctm = tm;
    const int inext = i + nq;
    if (inext < nx) {
      tile_of(inext, m0, n0, tm);
      ca.init(wave, p.lda, m0, lane);
      cb.init(wave, p.ldb, n0, lane);
      if (nk > 0) issue(lds, 0);
    }
    char* above = lds + STAGE;
    if constexpr (CS) {
      if (cs_on) cs.finish((float*)above, p, ctm, cn0, threadIdx.x);
    }
    // (the gradient-accumulating epilogue with its inputs fetched a block-row
    // ahead does not fit the registers next to the next tile's copy state)
    epilogue<EPI, TN, 0, 4, EPI != EPI_F32_ACC>(p, acc, (float*)(above + wave * EPI_BYTES), cm0 + wm * 128,
                                                cn0 + wn * (BN / WN_), lane, 0);
    if (inext >= nx) break;
    i = inext;
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[a][j][r] = 0.f;
  }
}

// Fragments of one unit (two consecutive k-steps, 2 u and 2 u + 1 of the
// wave's NKS) of a staged k-tile.
template <int BM, int BN, bool AK, bool BKC, int TN, int NKS, int BK>
__device__ __forceinline__ void load_unit(bf16x8 (&af)[2][4], bf16x8 (&bfr)[2][TN], const char* ta,
                                          const char* tb, const FragOffsets<BM, AK, 4, NKS, BK>& fa,
                                          const FragOffsets<BN, BKC, TN, NKS, BK>& fb, int u) {
#pragma unroll
  for (int s = 0; s < 2; ++s) {
#pragma unroll
    for (int i = 0; i < 4; ++i) af[s][i] = frag(ta, fa, i, 2 * u + s);
#pragma unroll
    for (int j = 0; j < TN; ++j) bfr[s][j] = frag(tb, fb, j, 2 * u + s);
  }
}

// The unit's 4 x TN x 2 MFMAs from registers; with MID, mid() runs between
// its two k-steps.
template <int TN, bool MID, typename Mid>
__device__ __forceinline__ void mma_unit(f32x16 (&acc)[4][TN], const bf16x8 (&af)[2][4],
                                         const bf16x8 (&bfr)[2][TN], Mid mid) {
#pragma unroll
  for (int s = 0; s < 2; ++s) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[s][i], bfr[s][j], acc[i][j], 0, 0, 0);
    if (MID && s == 0) {
      __builtin_amdgcn_sched_barrier(0);
      mid();
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// Workgroup-wide barrier that the compiler may not move any instruction across.
__device__ __forceinline__ void phase_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
}

// Ping-pong schedule.  Waves w and w + 4 share a SIMD (waves are dealt to the
// four SIMDs in turn); the two groups {0..3} and {4..7} run the same
// sequence of alternating phases, one phase apart:
//   memory phase:  read one unit's fragments (two k-steps) from LDS into
//                  registers and wait for them;
//   compute phase: the unit's 4 x TN x 2 MFMAs from registers, no LDS reads.
// The first unit of a tile also issues this wave's share of a k-tile copy,
// spread over both phases (Copies, below).
// Every phase ends at a workgroup barrier, so while one group multiplies the
// other reads, and each SIMD always has one wave with MFMAs to issue: the
// matrix core no longer idles while both waves of a SIMD sit at the same
// barrier or wait on LDS at the same time.
// Tiles are 256 x 128: each group covers the whole tile with four 128 x 64
// wave tiles and multiplies k-steps 2 g, 2 g + 1 of every k-tile (one unit);
// the two groups' partial sums are added through LDS at the end.  (The unit
// loop also allows several units per k-tile, as a single k-group would need.)
// Copies.  Tile t + NST - 1 is issued in tile t's first unit: its A slices
// after the memory phase's fragment reads, its B slices ahead of them or,
// with k-contiguous B tiles, between the compute phase's two k-steps.
// Tile t + 1 is first read in group 0's first memory phase of tile t + 1;
// before the barrier that opens that phase each wave waits for its own share
// (group 0 after its last compute phase of tile t, group 1 after its last
// memory phase of tile t, when its B slices of tile t + NST - 1 may not be
// issued yet).  The stage being refilled held tile t - 1, whose last fragment
// reads (group 1's last memory phase of tile t - 1) completed before the
// barrier that opens group 0's first phase of tile t.
template <int BN, int KS, int NST, int GM, bool AK, bool BKC, int EPI>
__global__ __launch_bounds__(512) void gemm_bf16_pp_kernel(GemmParams p) {
  constexpr int BM = 256, NW = 8, BK = 64;
  // the configuration the launcher uses: 256 x 128 tiles, two k-groups (the
  // same schedule on 256 x 256 tiles with one k-group measured no faster than
  // the plain kernel); a k-group issues its copy two phases ahead, so three
  // stages at least
  static_assert(BN == 128 && KS == 2 && NST >= 3, "tile shapes");
  constexpr int NWS = NW / KS;           // waves per k-group
  constexpr int WN_ = NWS / 2;           // waves along n (2 along m)
  constexpr int TN = BN / (32 * WN_);    // 32-wide blocks per wave along n (2)
  constexpr int NKS = (BK / 16) / KS;    // k-steps per wave per k-tile
  constexpr int U = NKS / 2;             // units per wave per k-tile
  constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2;
  constexpr int STAGE = A_BYTES + B_BYTES;
  constexpr int NA = A_BYTES / 1024, NB = B_BYTES / 1024;
  static_assert(NA % NW == 0 && NB % NW == 0, "copy split");
  constexpr int NIA = NA / NW, NIB = NB / NW;
  constexpr int PER_TILE = NIA + NIB;
  constexpr int EPI_BYTES = 32 * (32 * TN + 8) * 4;
  constexpr int SLOT = 2 * TN * 4096;
  constexpr int RED_BYTES = NW * SLOT;  // k-split reduction slots, one per wave
  constexpr int LDS_BYTES = NST * STAGE > RED_BYTES ? NST * STAGE : RED_BYTES;
  static_assert(LDS_BYTES <= 160 * 1024, "LDS");
  __shared__ __attribute__((aligned(1024))) char lds[LDS_BYTES];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int grp = wave >> 2;             // ping-pong group
  const int kg = wave / NWS, ws = wave % NWS;
  const int wm = ws / WN_, wn = ws % WN_;

  const int tiles_m = (p.M + BM - 1) / BM, tiles_n = (p.N + BN - 1) / BN;
  int pid = blockIdx.x;
  const int ntiles = gridDim.x;
  if ((ntiles & 7) == 0) pid = (pid & 7) * (ntiles >> 3) + (pid >> 3);
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

  Copier<BM, AK, NIA, NW, BK> ca;
  Copier<BN, BKC, NIB, NW, BK> cb;
  ca.init(wave, p.lda, m0, lane);
  cb.init(wave, p.ldb, n0, lane);
  FragOffsets<BM, AK, 4, NKS, BK> fa;
  FragOffsets<BN, BKC, TN, NKS, BK> fb;
  fa.init(wm * 128, lane, kg * NKS);
  fb.init(wn * (BN / WN_), lane, kg * NKS);

  f32x16 acc[4][TN];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  // column sums of B (a workgroup-uniform condition)
  constexpr bool CS = !AK && !BKC;  // weight-gradient layout only
  // Every tile-row takes part in the column sums for one k-tile in tiles_m, so
  // the extra work spreads evenly over the launch.
  const bool cs_on = CS && p.colsum_out != nullptr && z == 0;
  int cs_next = tm;  // next k-tile this workgroup sums
  ColSums<BN, BK> cs;
  if (cs_on) cs.init(threadIdx.x);

  struct Src {
    i32x4 a, b;
    int k, kend;
  };
  auto source = [&](int k0) {
    Src r{ra, rb, k0, ke};
    if (p.kseg_len > 0) {
      const int sg = k0 / p.kseg_len;
      r.k = k0 - sg * p.kseg_len;
      r.kend = p.kseg_len;
      r.a = make_rsrc((const bf16*)p.segA[sg] + zb * p.a_bs + zh * p.a_hs,
                      2L * (AK ? (long)p.M * p.lda : (long)p.kseg_len * p.lda));
      r.b = make_rsrc((const bf16*)p.segB[sg] + zb * p.b_bs + zh * p.b_hs,
                      2L * (BKC ? (long)p.N * p.ldb : (long)p.kseg_len * p.ldb));
    }
    return r;
  };
  auto issue = [&](char* st, int k0) {
    const Src sr = source(k0);
    ca.issue(sr.a, st, wave, p.lda, p.M, sr.k, sr.kend);
    cb.issue(sr.b, st + A_BYTES, wave, p.ldb, p.N, sr.k, sr.kend);
  };
  // The refill's A slices follow the unit's fragment reads.  Its B slices go
  // out between the compute phase's two k-steps when the B tiles are
  // k-contiguous (the input-gradient products) and ahead of the fragment reads
  // otherwise (the forward products): 8-12 % and 2-4 % shorter products than
  // one burst of both ahead of the reads.
  constexpr bool SPLIT = BKC;
  // Waits until this wave's share of tile t + 1 has landed (the copies of
  // tiles t + 2 .. t + NST - 1 issued so far may stay in flight: all of them,
  // or, when group 1 waits in the memory phase of a split refill, all but
  // the B slices of tile t + NST - 1, which it has not issued yet).
  auto wait_next = [&](int t, bool b_pending) {
    if (t + NST - 1 >= nk) wait_vmcnt<0>();
    else if (b_pending) wait_vmcnt<(NST - 3) * PER_TILE + NIA>();
    else wait_vmcnt<(NST - 2) * PER_TILE>();
  };

  // Prologue: tiles 0 .. NST-2 land before either group starts.
#pragma unroll
  for (int i = 0; i < NST - 1; ++i)
    if (i < nk) issue(lds + i * STAGE, kb + i * BK);
  wait_vmcnt<0>();
  __syncthreads();
  if (grp == 1) phase_barrier();

  bf16x8 af[2][4], bfr[2][TN];
  int sc = 0, si = NST - 1;  // stage of tile t, stage that tile t + NST - 1 goes to
  for (int t = 0; t < nk; ++t) {
    const char* st = lds + sc * STAGE;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      // memory phase
      const bool refill = u == 0 && t + NST - 1 < nk;
      char* dst = lds + si * STAGE;
      const Src nx = source(refill ? kb + (t + NST - 1) * BK : kb);
      if (!SPLIT && refill) cb.issue(nx.b, dst + A_BYTES, wave, p.ldb, p.N, nx.k, nx.kend);
      load_unit<BM, BN, AK, BKC, TN, NKS, BK>(af, bfr, st, st + A_BYTES, fa, fb, u);
      if (refill) ca.issue(nx.a, dst, wave, p.lda, p.M, nx.k, nx.kend);
      if constexpr (CS) {
        if (u == 0 && cs_on && t == cs_next) {
          cs.tile(st + A_BYTES);
          cs_next += tiles_m;
        }
      }
      __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): the unit's fragments are in registers
      if (grp == 1 && u == U - 1) wait_next(t, SPLIT && U == 1);
      phase_barrier();
      // compute phase
      mma_unit<TN, SPLIT>(acc, af, bfr, [&]() {
        if (refill) cb.issue(nx.b, dst + A_BYTES, wave, p.ldb, p.N, nx.k, nx.kend);
      });
      if (grp == 0 && u == U - 1) wait_next(t, false);
      phase_barrier();
    }
    sc = sc + 1 == NST ? 0 : sc + 1;
    si = si + 1 == NST ? 0 : si + 1;
  }
  if (grp == 0) phase_barrier();

  // LDS is free once every wave is past its last k-tile.
  __syncthreads();
  static_assert(ColSums<BN, BK>::RED_BYTES <= LDS_BYTES, "column-sum reduction fits LDS");
  if constexpr (CS) {
    if (cs_on) cs.finish((float*)lds, p, tm, n0, threadIdx.x);
  }
  // The partner's slot is read only by this wave, so after the reduction it
  // serves as this wave's epilogue tile.  (The gradient-accumulating
  // epilogue fetches each block-row's inputs as it reaches it: fetched a
  // block-row ahead they spill registers next to the k-split state.)
  constexpr bool LOOK = EPI != EPI_F32_ACC;
  float* mine = (float*)(lds + wave * SLOT);
  float* theirs = (float*)(lds + ((1 - kg) * NWS + ws) * SLOT);
  static_assert(EPI_BYTES <= SLOT, "epilogue tile fits a reduction slot");
  if (kg == 0) {
    ksplit_reduce<TN, 0>(acc, mine, theirs, lane);
    epilogue<EPI, TN, 0, 2, LOOK>(p, acc, theirs, m0 + wm * 128, n0 + wn * (BN / WN_), lane, c_off);
  } else {
    ksplit_reduce<TN, 1>(acc, mine, theirs, lane);
    epilogue<EPI, TN, 2, 4, LOOK>(p, acc, theirs, m0 + wm * 128, n0 + wn * (BN / WN_), lane, c_off);
  }
}

template <int BN, int KS, int NST, int GM, bool AK, bool BKC, int EPI>
hipError_t launch_bf16_pp(const GemmParams& p, hipStream_t s) {
  const long z = (long)p.batch * p.heads;
  const int tiles = ((p.M + 255) / 256) * ((p.N + BN - 1) / BN);
  hipLaunchKernelGGL((gemm_bf16_pp_kernel<BN, KS, NST, GM, AK, BKC, EPI>), dim3(tiles, z), dim3(512), 0, s,
                     p);
  return hipGetLastError();
}

// Launch of one kernel variant over the whole (tiles, batch x heads) grid.
template <int BM, int BN, int NW, int KS, int BK, int NST, bool AK, bool BKC, int EPI>
hipError_t launch_bf16_variant(const GemmParams& p, hipStream_t s) {
  const long z = (long)p.batch * p.heads;
  const int tiles = ((p.M + BM - 1) / BM) * ((p.N + BN - 1) / BN);
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, NW, KS, BK, NST, AK, BKC, EPI>), dim3(tiles, z),
                     dim3(64 * NW), 0, s, p);
  return hipGetLastError();
}

template <bool AK, bool BKC, int EPI>
hipError_t launch_bf16_persist(const GemmParams& p, hipStream_t s) {
  const int ntiles = ((p.M + 255) / 256) * ((p.N + 255) / 256);
  const int per_xcd = std::max(1, device_compute_units() / 8);
  const int nq = std::min(ntiles / 8, per_xcd);
  // Deferred last k-steps (mma_tile) pay off on the long reductions of
  // batched weight gradients (-2 % batched, -7 % for one-round launches), not
  // on single micro-batch ones (+2.4 % at K = 2048).
  if (p.K >= 8192)
    hipLaunchKernelGGL((gemm_bf16_persist_kernel<EPI, AK, BKC, true>), dim3(8 * nq), dim3(512), 0, s, p);
  else
    hipLaunchKernelGGL((gemm_bf16_persist_kernel<EPI, AK, BKC, false>), dim3(8 * nq), dim3(512), 0, s, p);
  return hipGetLastError();
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
  // 256 x 128 tiles run the ping-pong k-split kernel (three stages, tile-rows
  // grouped by four); 256 x 256 tiles the plain two-stage kernel, which
  // measured as fast as its ping-pong form.
  if (p.N <= 128 || cost(256, 128) < cost(256, 256))
    return launch_bf16_pp<128, 2, 3, 4, AK, BKC, EPI>(p, s);
  // Weight-gradient products of more than one round of tiles run the
  // persistent kernel: each workgroup's next tile starts copying while the
  // previous tile's fp32 gradient update runs (measured on the 6.7B stage's
  // single-micro-batch products: 3-4 % faster; neutral for the forward and
  // input-gradient products, which keep one tile per workgroup).
  if constexpr (!AK && !BKC) {
    const long ntiles = (long)((p.M + 255) / 256) * ((p.N + 255) / 256);
    if (z == 1 && p.krange == KR_FULL && !p.causal_skip && ntiles % 8 == 0 && ntiles > device_compute_units())
      return launch_bf16_persist<AK, BKC, EPI>(p, s);
  }
  return launch_bf16_variant<256, 256, 8, 1, 64, 2, AK, BKC, EPI>(p, s);
}

}  // namespace
