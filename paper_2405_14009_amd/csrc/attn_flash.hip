// Fused attention core for bf16 stages with head dimension 128, on CDNA4
// matrix cores (v_mfma_f32_32x32x16_bf16, fp32 accumulate).  Computes the
// attention of the GPT block (Sec. 5 model family): per (sequence, head)
// S = Q K^T / sqrt(d), causal mask, P = softmax(S), O = P V, and its input
// gradient, without materialising S or P in memory:
//
//   forward   one pass over key blocks with a running row maximum and row sum
//             (the softmax is rescaled as the maximum grows); O and the row
//             log-sum-exp (base 2, of the scaled scores) are written.
//   backward  P is recomputed from Q, K and the stored log-sum-exp;
//             Dv = rowsum(dO o O) (= rowsum(dP o P));  dS = P o (dP - Dv);
//             dQ = scale dS K, and Dv (kernel over query blocks, first), then
//             dV = P^T dO, dK = scale dS^T Q (kernel over key blocks).
//             Two kernels instead of atomics keep every sum in a fixed order,
//             so the result is bitwise reproducible.
//
// Operand layout.  Q, K, V are the column blocks [Q | K | V] of the [T, 3h]
// projection output (head j at columns j*128 of each block); O and dO are
// [T, h] with head j at columns j*128; dQ, dK, dV are written into the same
// three column blocks of the [T, 3h] gradient.
//
// MFMA layout (32x32x16): A fragment: lane l holds row l % 32, k = 8 (l / 32)
// + 0..7; B fragment: column l % 32, same k; result: lane l holds column
// l % 32, rows 8 (r / 4) + 4 (l / 32) + r % 4 (r = 0..15).  The kernels
// arrange every product so that the score block comes out with one query (or
// one key) per lane column: softmax statistics are then per lane, and the
// score registers are directly the B fragment of the next product when the
// k positions of that product are mapped to
//   k = 8 (l / 32) + e  ->  token 4 (l / 32) + (e % 4) + 8 (e / 4)
// within each 16-token step; the A fragments of that product are read with
// ds_read_b64_tr_b16 at matching token rows.
//
// Tiles of [rows][128] bf16 (256 bytes per row) are staged in LDS by
// buffer-load-to-LDS copies, 16-byte chunk c of row r stored at chunk
// c ^ swz(r), swz(r) = 4 (r % 4) + (r / 4) % 4: both the row reads
// (ds_read_b128, 16 consecutive rows of one chunk) and the transposing reads
// (ds_read_b64_tr_b16, 4 consecutive rows of 4 chunks) are free of bank
// conflicts.
#include <cmath>

#include "common.h"
#include "kernels.h"
#include "mfma_common.h"

namespace {

constexpr int HD = 128;          // head dimension
constexpr int ROWB = 2 * HD;     // bytes per tile row
constexpr int TILE64 = 64 * ROWB;  // bytes of a 64-row tile
constexpr float kLog2e = 1.4426950408889634f;

struct AttnArgs {
  const bf16* qkv;  // [b*s, 3h]
  const bf16* o;    // [b*s, h]
  const bf16* dout; // [b*s, h]
  bf16* out;        // forward: O [b*s, h];  backward: dQKV [b*s, 3h]
  float* lse;       // [b, heads, s]  base-2 log-sum-exp of the scaled scores
  float* dv;        // [b, heads, s]  rowsum(dO o O)
  int s, heads, bh, h;
  float scale, sl2;  // 1/sqrt(d), 1/sqrt(d) * log2(e)
};

__device__ __forceinline__ int swz(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }

// This wave's share of the copy of a [ROWS][128] tile: rows row0.. of a
// row-major matrix (leading dimension ld elements, rows >= nrows read as
// zeros).  Slice g (1 KB = 4 rows) is copied by wave g % 4.
template <int ROWS>
__device__ __forceinline__ void load_tile(const i32x4& rs, char* tile, int wave, int lane, long ld,
                                          int row0, int nrows) {
  const int c = (lane & 15) ^ ((((lane >> 4) & 3) << 2) | wave);
#pragma unroll
  for (int j = 0; j < ROWS / 16; ++j) {
    const int gr = row0 + 4 * wave + 16 * j + (lane >> 4);
    const uint32_t off = gr < nrows ? (uint32_t)gr * (uint32_t)(2 * ld) + 16u * c : kOOB;
    dma16(rs, __builtin_amdgcn_readfirstlane(lds_addr(tile) + (wave + 4 * j) * 1024), off);
  }
}

// 64 floats (one per row of a 64-row block, rows >= nrows as zeros) into a
// 1 KB LDS area; issued by one wave.
__device__ __forceinline__ void load_vec64(const i32x4& rs, char* dst, int lane, int row0, int nrows) {
  const int r = row0 + 4 * lane;
  const uint32_t off = (lane < 16 && r < nrows) ? 4u * r : kOOB;
  dma16(rs, __builtin_amdgcn_readfirstlane(lds_addr(dst)), off);
}

// Warm L2 with 32 rows (row0.., rows >= nrows skipped) of a row-major bf16
// matrix with 128-column rows: eight copies of 4 rows into a 1 KB LDS sink
// that nothing reads.  Issued a step before the rows are loaded into
// registers, so that load hits L2 instead of waiting on HBM.
__device__ __forceinline__ void warm_rows32(const i32x4& rs, char* sink, int lane, long ld, int row0,
                                            int nrows) {
  const int c = lane & 15;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int gr = row0 + 4 * j + (lane >> 4);
    const uint32_t off = gr < nrows ? (uint32_t)gr * (uint32_t)(2 * ld) + 16u * c : kOOB;
    dma16(rs, __builtin_amdgcn_readfirstlane(lds_addr(sink)), off);
  }
}

// Row read: 32-row block starting at row 0 of the tile, k-step ks (16 of the
// 128 columns): lane l gets row l % 32, columns 16 ks + 8 (l / 32) + 0..7.
struct RowOffs {
  uint32_t off[HD / 16];
  __device__ __forceinline__ void init(int lane) {
    const int r = lane & 31;
#pragma unroll
    for (int ks = 0; ks < HD / 16; ++ks) off[ks] = r * ROWB + (((2 * ks + (lane >> 5)) ^ swz(r)) << 4);
  }
};
__device__ __forceinline__ bf16x8 rd_row(const char* tile, const RowOffs& o, int blk, int ks) {
  return *(const bf16x8*)(tile + o.off[ks] + blk * 32 * ROWB);
}

// Transposing read: columns 32 dblk + (l % 32) of the tile as rows (m), tile
// rows as k: lane l gets tile rows 16 t + 4 (l / 32) + {0..3, 8..11}.
struct TrOffs {
  uint32_t off[HD / 32][2];
  __device__ __forceinline__ void init(int lane) {
    const int i = lane & 15, g = (lane >> 4) & 1, hh = lane >> 5;
#pragma unroll
    for (int b = 0; b < HD / 32; ++b)
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int r = 4 * hh + (i >> 2) + 8 * half;
        const int c = 4 * b + 2 * g + ((i & 3) >> 1);
        off[b][half] = r * ROWB + ((c ^ swz(r)) << 4) + 8 * (i & 1);
      }
  }
};
__device__ __forceinline__ bf16x8 rd_tr(const char* tile, const TrOffs& o, int dblk, int t) {
  const char* p0 = tile + o.off[dblk][0] + t * 16 * ROWB;
  const char* p1 = tile + o.off[dblk][1] + t * 16 * ROWB;
  s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)p0);
  s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)p1);
  s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ f32x16 mfma(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Two independent MFMA chains over the head dimension: a0 += rows of block
// b0 of tile t0 times s0, a1 += rows of block b1 of tile t1 times s1 (the
// stationary operands in registers).  The fragments of k-step ks + D are read
// while the MFMAs of ks issue, so LDS latency hides behind D k-steps of
// matrix work instead of stalling every step.
template <int D>
__device__ __forceinline__ void two_chains(f32x16& a0, const char* t0, int b0, const bf16x8 (&s0)[HD / 16],
                                           f32x16& a1, const char* t1, int b1, const bf16x8 (&s1)[HD / 16],
                                           const RowOffs& ro) {
  constexpr int NK = HD / 16, NB = D + 1;
  bf16x8 f[NB][2];
#pragma unroll
  for (int i = 0; i < D; ++i) {
    f[i][0] = rd_row(t0, ro, b0, i);
    f[i][1] = rd_row(t1, ro, b1, i);
  }
  // scheduling groups pin the order (otherwise the scheduler sinks each read
  // next to its MFMA to save registers): D k-steps of reads, then per k-step
  // the next reads followed by this step's two MFMAs
  __builtin_amdgcn_sched_group_barrier(0x100, 2 * D, 0);
#pragma unroll
  for (int ks = 0; ks < NK; ++ks) {
    if (ks + D < NK) {
      f[(ks + D) % NB][0] = rd_row(t0, ro, b0, ks + D);
      f[(ks + D) % NB][1] = rd_row(t1, ro, b1, ks + D);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
    a0 = mfma(f[ks % NB][0], s0[ks], a0);
    a1 = mfma(f[ks % NB][1], s1[ks], a1);
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
  }
}

// B fragment of 16-token step t from a pair of score blocks (32 tokens each):
// elements r = 8 (t % 2) .. +7 of block t / 2, rounded to bf16.
__device__ __forceinline__ bf16x8 pack_frag(const f32x16 (&p)[2], int t) {
  bf16x8 v;
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = (bf16)p[t >> 1][8 * (t & 1) + e];
  return v;
}

// B fragment of the 16-token step `half` of one score block (32 tokens).
__device__ __forceinline__ bf16x8 pack_half(const f32x16& p, int half) {
  bf16x8 v;
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = (bf16)p[8 * half + e];
  return v;
}

// Global 16-byte fragment of a stationary operand: row `row` (zeros when
// row >= nrows), columns 16 ks + 8 (l / 32) + 0..7.
__device__ __forceinline__ void load_stationary(bf16x8 (&f)[HD / 16], const bf16* base, long ld, int row,
                                                int nrows, int lane) {
#pragma unroll
  for (int ks = 0; ks < HD / 16; ++ks) {
    if (row < nrows) {
      f[ks] = *(const bf16x8*)(base + (long)row * ld + 16 * ks + 8 * (lane >> 5));
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) f[ks][e] = (bf16)0.f;
    }
  }
}

// Wait for every outstanding vector memory access of this wave.  Used after
// loads on a rarely taken branch: the compiler otherwise carries them as
// pending into the code after the branch and waits for them there on every
// path, which also waits for the tile copies issued in between.
__device__ __forceinline__ void vm_drain() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Store a [128 (d) x 32 (tokens)] accumulator set (result layout: lane column
// = token, rows = d) as rows of a row-major bf16 matrix: 8-byte pieces.
__device__ __forceinline__ void store_dT(const f32x16 (&acc)[HD / 32], bf16* base, long ld, int row,
                                         int nrows, int lane, float mul) {
  if (row >= nrows) return;
  bf16* p = base + (long)row * ld + 4 * (lane >> 5);
#pragma unroll
  for (int b = 0; b < HD / 32; ++b)
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      bf16 t[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) t[e] = (bf16)(acc[b][4 * rg + e] * mul);
      *(uint2*)(p + 32 * b + 8 * rg) = *(const uint2*)t;
    }
}

// The same block through this wave's 8 KB of LDS (t): rows written as bf16
// (16-byte chunk c of row r at chunk c ^ (r % 16), so the 32 rows of one
// write land on distinct banks), then read back 16 bytes per lane, so each
// store instruction writes four whole 256-byte rows instead of 16-byte pieces
// of 32 rows.  row0 is the wave's first row (lane l holds row row0 + l % 32).
// The LDS accesses of one wave complete in order, so no wait is needed
// between the two halves.
__device__ __forceinline__ void store_rows_lds(const f32x16 (&acc)[HD / 32], char* t, bf16* base, long ld,
                                               int row0, int nrows, int lane, float mul) {
  const int r = lane & 31, hf = lane >> 5;
#pragma unroll
  for (int b = 0; b < HD / 32; ++b)
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      bf16 v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = (bf16)(acc[b][4 * rg + e] * mul);
      const int c = 4 * b + rg;  // columns 32 b + 8 rg + 4 hf + e
      *(uint2*)(t + r * ROWB + ((c ^ (r & 15)) << 4) + 8 * hf) = *(const uint2*)v;
    }
  const int c = lane & 15;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int rr = 4 * i + (lane >> 4);
    const uint4 v = *(const uint4*)(t + rr * ROWB + ((c ^ (rr & 15)) << 4));
    if (row0 + rr < nrows) *(uint4*)(base + (long)(row0 + rr) * ld + 8 * c) = v;
  }
}

__device__ __forceinline__ void zero(f32x16& a) {
#pragma unroll
  for (int r = 0; r < 16; ++r) a[r] = 0.f;
}

// Workgroup -> (sequence*head z, block index) with the longest blocks first.
__device__ __forceinline__ void block_of(const AttnArgs& p, int nblk, bool longest_last_index, int& z,
                                         int& blk) {
  const int x = blockIdx.x;
  z = x % p.bh;
  const int q = x / p.bh;
  blk = longest_last_index ? nblk - 1 - q : q;
}

// ---------------------------------------------------------------------------
// Forward.  Per wave: 32 queries (lane column = query), Q rows stationary in
// registers; key blocks of 64 staged in LDS (K and V).  Per wave and key
// block: S^T = K Q^T (16 MFMAs), online softmax per lane (= per query),
// O^T += V^T P^T (16 MFMAs).

// Online-softmax state of a wave's 32 queries: unnormalised O^T, the
// reference maximum (base-2 scaled score units) and this lane's share of the
// row sum (lanes l and l + 32 hold the two halves of each key block's rows).
struct FwdState {
  f32x16 o[HD / 32];
  float m_run, l_run;
  // The first key block a query takes part in always moves the reference
  // maximum, and every query's row keeps its diagonal key.
  __device__ __forceinline__ void reset() {
#pragma unroll
    for (int b = 0; b < HD / 32; ++b) zero(o[b]);
    m_run = -1e30f;
    l_run = 0.f;
  }
};

// Key masking of a score block whose lane column is a query (lane l: query
// qq = q0 + l % 32).  Element r of 32-key half j holds key
//   k0 + 32 j + 4 (l / 32) + kofs(r),  kofs(r) = 8 (r / 4) + r % 4,
// which is masked when it lies past the sequence end or, causal, after qq,
// i.e. when 32 j + kofs(r) > key_room = min(qq (causal), s - 1) - k0 - 4 (l / 32):
// one compare per element against a constant.  Callers take this path only
// for the blocks that straddle the diagonal or the sequence end.
__device__ __forceinline__ constexpr int kofs(int r) { return 8 * (r >> 2) + (r & 3); }
template <bool CAUSAL>
__device__ __forceinline__ int key_room(int k0, int qq, int lane, const AttnArgs& p) {
  const int last = CAUSAL ? min(qq, p.s - 1) : p.s - 1;
  return last - k0 - 4 * (lane >> 5);
}
// A wave-uniform condition as such for the compiler (its operands are
// uniform, but the compiler cannot always tell): the masking then stays a
// branch that only the blocks needing it take, instead of selects that
// every block executes.
__device__ __forceinline__ bool uniform(bool c) { return __builtin_amdgcn_readfirstlane((int)c) != 0; }
template <int NJ>
__device__ __forceinline__ void mask_scores(f32x16 (&sc)[NJ], int room, float v) {
#pragma unroll
  for (int j = 0; j < NJ; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (32 * j + kofs(r) > room) sc[j][r] = v;
}

// One key block (keys k0..k0+63; K tile kt, V tile vt) for the wave's queries
// q0..q0+31 (this lane's query qq).
template <bool CAUSAL>
__device__ __forceinline__ void fwd_block(FwdState& st, const bf16x8 (&qf)[HD / 16], const char* kt,
                                          const char* vt, const RowOffs& ro, const TrOffs& to, int k0,
                                          int q0, int qq, int lane, const AttnArgs& p) {
  if (CAUSAL && k0 > q0 + 31) return;  // every key of the block is after every query of the wave
  f32x16 sc[2];
  zero(sc[0]);
  zero(sc[1]);
  two_chains<2>(sc[0], kt, 0, qf, sc[1], kt, 1, qf, ro);
  // Masked keys (past the sequence end or, causal, after the query) at -inf.
  if (uniform((CAUSAL && k0 + 63 > q0) || k0 + 64 > p.s))
    mask_scores<2>(sc, key_room<CAUSAL>(k0, qq, lane, p), -INFINITY);
  // Row maximum over the raw scores (the scale is positive); the scale is
  // folded into the exponent's FMA below.
  float mx = -INFINITY;
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[j][r]);
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * p.sl2;
  // Lazy rescaling: the reference maximum moves only when a row's maximum
  // exceeds it by more than 8 (base 2), so most key blocks skip rescaling O
  // and the row sum.  Exponentials are then at most 2^8, and O / l and the
  // log-sum-exp are unchanged in exact arithmetic.
  const bool grow = mx > st.m_run + 8.f;
  if (__any(grow)) {
    const float m_new = grow ? mx : st.m_run;
    const float alpha = __builtin_amdgcn_exp2f(st.m_run - m_new);
    st.m_run = m_new;
    st.l_run *= alpha;
#pragma unroll
    for (int b = 0; b < HD / 32; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) st.o[b][r] *= alpha;
  }
  float ls = 0.f;
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float e = __builtin_amdgcn_exp2f(fmaf(sc[j][r], p.sl2, -st.m_run));
      sc[j][r] = e;
      ls += e;
    }
  st.l_run += ls;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const bf16x8 pf = pack_frag(sc, t);
#pragma unroll
    for (int b = 0; b < HD / 32; ++b) st.o[b] = mfma(rd_tr(vt, to, b, t), pf, st.o[b]);
  }
}

// O = O~ / l and the row log-sum-exp m + log2 l of the wave's queries
// q0..q0+31 (this lane's qq); through LDS area t (8 KB) when given.
__device__ __forceinline__ void fwd_store(const FwdState& st, const AttnArgs& p, int z, int q0, int qq,
                                          int lane, char* t = nullptr) {
  const int zb = z / p.heads, zh = z % p.heads;
  const float l_tot = st.l_run + __shfl_xor(st.l_run, 32, 64);
  const float inv = 1.0f / l_tot;
  bf16* const out = (bf16*)p.out + (long)zb * p.s * p.h + zh * HD;
  if (t)
    store_rows_lds(st.o, t, out, p.h, q0, p.s, lane, inv);
  else
    store_dT(st.o, out, p.h, qq, p.s, lane, inv);
  if (lane < 32 && qq < p.s) p.lse[(long)z * p.s + qq] = st.m_run + __builtin_amdgcn_logf(l_tot);
}

// One query block of 128 per workgroup (4 waves), two stages of K and V.
template <bool CAUSAL>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_fwd_k(AttnArgs p) {
  __shared__ __attribute__((aligned(1024))) char lds0[2 * TILE64];
  __shared__ __attribute__((aligned(1024))) char lds1[2 * TILE64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nqb = (p.s + 127) / 128;
  int z, qb;
  block_of(p, nqb, CAUSAL, z, qb);
  const int zb = z / p.heads, zh = z % p.heads;
  const long ld = 3L * p.h;
  const bf16* Q = p.qkv + (long)zb * p.s * ld + zh * HD;
  const i32x4 rk = make_rsrc(Q + p.h, 2L * p.s * ld);
  const i32x4 rv = make_rsrc(Q + 2 * p.h, 2L * p.s * ld);
  const int q0 = qb * 128 + 32 * wave;
  const int qq = q0 + (lane & 31);

  bf16x8 qf[HD / 16];
  load_stationary(qf, Q, ld, qq, p.s, lane);
  RowOffs ro;
  ro.init(lane);
  TrOffs to;
  to.init(lane);
  FwdState st;
  st.reset();

  const int nkb_all = (p.s + 63) / 64;
  const int nkb = CAUSAL ? min(nkb_all, 2 * qb + 2) : nkb_all;

  auto issue = [&](char* t, int kb) {
    load_tile<64>(rk, t, wave, lane, ld, kb * 64, p.s);
    load_tile<64>(rv, t + TILE64, wave, lane, ld, kb * 64, p.s);
  };
  auto compute = [&](const char* t, int kb) {
    fwd_block<CAUSAL>(st, qf, t, t + TILE64, ro, to, kb * 64, q0, qq, lane, p);
  };

  if (nkb > 0) issue(lds0, 0);
  stage_sync();
  int kb = 0;
  for (; kb + 1 < nkb; kb += 2) {
    issue(lds1, kb + 1);
    compute(lds0, kb);
    stage_sync();
    if (kb + 2 < nkb) issue(lds0, kb + 2);
    compute(lds1, kb + 1);
    stage_sync();
  }
  if (kb < nkb) compute(lds0, kb);
  __syncthreads();  // every wave is done with the tiles: lds0 holds the output rows
  fwd_store(st, p, z, q0, qq, lane, lds0 + wave * 32 * ROWB);
}

// Causal forward over pairs of query blocks.  Query block q needs the key
// blocks [0, n(q)), n(q) = min(ceil(s / 64), 2 q + 2): at s = 2048 the first
// and the last block differ 16-fold in work, and with one block per
// workgroup some SIMDs idle while others finish long blocks.  Here a
// workgroup of eight waves takes the blocks qa = i and qb = nqb - 1 - i
// (n(qa) + n(qb) is about the same for every pair) and cuts the sequence of
// steps [qa: key blocks 0..n(qa)), [qb: key blocks 0..n(qb)) in two halves:
// waves 0-3 run the first half (all of qa, then the first key blocks of qb),
// waves 4-7 the rest of qb.  Waves w and w + 4 share a SIMD, so every SIMD
// carries half of the pair.  The two partial softmax states of qb (lane for
// lane the same queries) are merged through LDS at the end.  A middle block
// (odd nqb) pairs with itself: its key blocks are split the same way.
constexpr int FWD_STAGE = 2 * TILE64;        // K | V of one key block
constexpr int FWD_GROUP = 2 * FWD_STAGE;     // two stages per wave group

__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_fwd_pair_k(AttnArgs p) {
  // [group 0 stages | group 1 stages | L2-warming sink | merge statistics];
  // after the loop the stages hold group 0's partial O (first 64 KB) and the
  // output rows on their way to memory (the next 64 KB), so the statistics
  // the merge reads have an area of their own
  __shared__ __attribute__((aligned(1024))) char lds[2 * FWD_GROUP + 1024 + 2048];
  char* const sink = lds + 2 * FWD_GROUP;
  float2* const mstat = (float2*)(lds + 2 * FWD_GROUP + 1024);  // qb's (maximum, sum) per [wave][lane]
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int grp = wave >> 2, wg = wave & 3;
  const int nqb = (p.s + 127) / 128;
  const int z = blockIdx.x % p.bh, pr = blockIdx.x / p.bh;
  const int qa = pr, qb = nqb - 1 - pr;
  const int nkb_all = (p.s + 63) / 64;
  const int nb = min(nkb_all, 2 * qb + 2);
  const int na = qa == qb ? 0 : min(nkb_all, 2 * qa + 2);
  const int half = (na + nb + 1) / 2;
  const int j0 = grp ? half : 0;                     // this group's first step
  const int cnt = grp ? na + nb - half : half;       // and its number of steps
  const int zb = z / p.heads, zh = z % p.heads;
  const long ld = 3L * p.h;
  const bf16* Q = p.qkv + (long)zb * p.s * ld + zh * HD;
  const i32x4 rk = make_rsrc(Q + p.h, 2L * p.s * ld);
  const i32x4 rv = make_rsrc(Q + 2 * p.h, 2L * p.s * ld);
  const i32x4 rq = make_rsrc(Q, 2L * p.s * ld);

  int qcur = j0 < na ? qa : qb;
  int q0 = qcur * 128 + 32 * wg;
  int qq = q0 + (lane & 31);
  bf16x8 qf[HD / 16];
  load_stationary(qf, Q, ld, qq, p.s, lane);
  // fragment offsets carry the group's LDS base, so stage pointers stay constants
  RowOffs ro;
  ro.init(lane);
  TrOffs to;
  to.init(lane);
#pragma unroll
  for (int ks = 0; ks < HD / 16; ++ks) ro.off[ks] += grp * FWD_GROUP;
#pragma unroll
  for (int b = 0; b < HD / 32; ++b) {
    to.off[b][0] += grp * FWD_GROUP;
    to.off[b][1] += grp * FWD_GROUP;
  }
  FwdState st;
  st.reset();

  auto key_block = [&](int j) { return j < na ? j : j - na; };
  auto issue = [&](char* t, int j) {
    char* g = t + grp * FWD_GROUP;
    const int kb = key_block(j);
    load_tile<64>(rk, g, wg, lane, ld, kb * 64, p.s);
    load_tile<64>(rv, g + TILE64, wg, lane, ld, kb * 64, p.s);
  };
  // step it of this group: (on moving to qb, its Q rows first, so the first
  // products wait for them and not for the copy), the copy of the next step's
  // tiles, then the products
  auto step = [&](int it, const char* cur, char* nxt) {
    const int j = j0 + it;
    if (it < cnt && j == na && qcur != qb) {  // group 0 leaves qa: its rows are complete
      fwd_store(st, p, z, q0, qq, lane);
      st.reset();
      qcur = qb;
      q0 = qcur * 128 + 32 * wg;
      qq = q0 + (lane & 31);
      load_stationary(qf, Q, ld, qq, p.s, lane);
      vm_drain();
    }
    if (it < cnt && j + 1 == na) warm_rows32(rq, sink, lane, ld, qb * 128 + 32 * wg, p.s);
    if (it + 1 < cnt) issue(nxt, j + 1);
    if (it < cnt) fwd_block<true>(st, qf, cur, cur + TILE64, ro, to, key_block(j) * 64, q0, qq, lane, p);
  };

  if (cnt > 0) issue(lds, j0);
  stage_sync();
  int it = 0;
  for (; it + 1 < half; it += 2) {
    step(it, lds, lds + FWD_STAGE);
    stage_sync();
    step(it + 1, lds + FWD_STAGE, lds);
    stage_sync();
  }
  if (it < half) {
    step(it, lds, lds + FWD_STAGE);
    stage_sync();
  }

  // Merge qb: group 0 publishes its partial state (lane-major float4 chunks,
  // conflict-free), group 1 combines it with its own and stores.
  if (grp == 0) {
    if (qcur != qb) {  // no step of qb in this half: qa is complete, qb's share is empty
      fwd_store(st, p, z, q0, qq, lane, lds + FWD_GROUP + 4 * 32 * ROWB + wg * 32 * ROWB);
      st.reset();
    }
    float4* dst = (float4*)lds + wg * 16 * 64 + lane;
#pragma unroll
    for (int b = 0; b < HD / 32; ++b)
#pragma unroll
      for (int c = 0; c < 4; ++c)
        dst[(4 * b + c) * 64] = make_float4(st.o[b][4 * c], st.o[b][4 * c + 1], st.o[b][4 * c + 2],
                                            st.o[b][4 * c + 3]);
    mstat[wg * 64 + lane] = make_float2(st.m_run, st.l_run);
  }
  __syncthreads();
  if (grp == 1) {
    const float2 ml = mstat[wg * 64 + lane];
    const float m = fmaxf(ml.x, st.m_run);
    const float a0 = __builtin_amdgcn_exp2f(ml.x - m), a1 = __builtin_amdgcn_exp2f(st.m_run - m);
    const float4* src = (const float4*)lds + wg * 16 * 64 + lane;
#pragma unroll
    for (int b = 0; b < HD / 32; ++b)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const float4 v = src[(4 * b + c) * 64];
        st.o[b][4 * c] = v.x * a0 + st.o[b][4 * c] * a1;
        st.o[b][4 * c + 1] = v.y * a0 + st.o[b][4 * c + 1] * a1;
        st.o[b][4 * c + 2] = v.z * a0 + st.o[b][4 * c + 2] * a1;
        st.o[b][4 * c + 3] = v.w * a0 + st.o[b][4 * c + 3] * a1;
      }
    st.l_run = ml.y * a0 + st.l_run * a1;
    st.m_run = m;
    fwd_store(st, p, z, q0, qq, lane, lds + FWD_GROUP + wg * 32 * ROWB);
  }
}

// ---------------------------------------------------------------------------
// Backward over key blocks: dK, dV.  Workgroup: 128 keys of one (sequence,
// head), 4 waves x 32 keys (K and V rows stationary in registers); query
// blocks of 64 staged in LDS (Q, dO, log-sum-exp and Dv; two stages).  Per
// wave and query block: S = Q K^T and dP = dO V^T (lane column = key),
// P = exp2(S sl2 - lse), dS = P (dP - Dv); dV^T += dO^T P, dK^T += Q^T dS.
template <bool CAUSAL>
__global__ __launch_bounds__(256) void attn_bwd_kv_k(AttnArgs p) {
  constexpr int STAGE = 2 * TILE64 + 2048;
  __shared__ __attribute__((aligned(1024))) char lds0[STAGE];
  __shared__ __attribute__((aligned(1024))) char lds1[STAGE];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nkb = (p.s + 127) / 128;
  int z, kb;
  block_of(p, nkb, false, z, kb);
  const int zb = z / p.heads, zh = z % p.heads;
  const long ld = 3L * p.h;
  const bf16* Q = p.qkv + (long)zb * p.s * ld + zh * HD;
  const bf16* K = Q + p.h;
  const bf16* V = Q + 2 * p.h;
  const bf16* dO = p.dout + (long)zb * p.s * p.h + zh * HD;
  const i32x4 rq = make_rsrc(Q, 2L * p.s * ld);
  const i32x4 rdo = make_rsrc(dO, 2L * p.s * p.h);
  const i32x4 rl = make_rsrc(p.lse + (long)z * p.s, 4L * p.s);
  const i32x4 rd = make_rsrc(p.dv + (long)z * p.s, 4L * p.s);
  const int k0w = kb * 128 + 32 * wave;
  const int key = k0w + (lane & 31);

  bf16x8 kf[HD / 16], vf[HD / 16];
  load_stationary(kf, K, ld, key, p.s, lane);
  load_stationary(vf, V, ld, key, p.s, lane);
  RowOffs ro;
  ro.init(lane);
  TrOffs to;
  to.init(lane);

  f32x16 dk[HD / 32], dv[HD / 32];
#pragma unroll
  for (int b = 0; b < HD / 32; ++b) {
    zero(dk[b]);
    zero(dv[b]);
  }
  const int nqb_all = (p.s + 63) / 64;
  const int qb0 = CAUSAL ? 2 * kb : 0;

  auto issue = [&](char* st, int qb) {
    load_tile<64>(rq, st, wave, lane, ld, qb * 64, p.s);
    load_tile<64>(rdo, st + TILE64, wave, lane, p.h, qb * 64, p.s);
    if (wave == 0) load_vec64(rl, st + 2 * TILE64, lane, qb * 64, p.s);
    if (wave == 1) load_vec64(rd, st + 2 * TILE64 + 1024, lane, qb * 64, p.s);
  };
  auto compute = [&](const char* st, int qb) {
    const int qs = qb * 64;
    if (CAUSAL && qs + 63 < k0w) return;  // every query of the block precedes every key of the wave
    const char* qt = st;
    const char* ot = st + TILE64;
    const float* lse = (const float*)(st + 2 * TILE64);
    const float* dvv = (const float*)(st + 2 * TILE64 + 1024);
    const bool need_mask = uniform(CAUSAL && qs < k0w + 31);
    // the two 32-query halves of the block in turn (one half's scores live)
#pragma unroll 1
    for (int j = 0; j < 2; ++j) {
      f32x16 sc, dp;
      zero(sc);
      zero(dp);
      two_chains<2>(sc, qt, j, kf, dp, ot, j, vf, ro);
      float Dv[16];
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const int ql = 32 * j + 8 * rg + 4 * (lane >> 5);
        const float4 L4 = *(const float4*)(lse + ql);
        const float4 D4 = *(const float4*)(dvv + ql);
        const float Lv[4] = {L4.x, L4.y, L4.z, L4.w};
        Dv[4 * rg] = D4.x;
        Dv[4 * rg + 1] = D4.y;
        Dv[4 * rg + 2] = D4.z;
        Dv[4 * rg + 3] = D4.w;
#pragma unroll
        for (int e = 0; e < 4; ++e) sc[4 * rg + e] = __builtin_amdgcn_exp2f(sc[4 * rg + e] * p.sl2 - Lv[e]);
      }
      // element r holds query qs + 32 j + 4 (l / 32) + kofs(r): masked when
      // that query precedes this lane's key
      if (need_mask) {
        const int room = key - qs - 32 * j - 4 * (lane >> 5);
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (kofs(r) < room) sc[r] = 0.f;
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) dp[r] = sc[r] * (dp[r] - Dv[r]);
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const int t = 2 * j + hf;
        const bf16x8 pf = pack_half(sc, hf);
        const bf16x8 sf = pack_half(dp, hf);
#pragma unroll
        for (int b = 0; b < HD / 32; ++b) {
          dv[b] = mfma(rd_tr(ot, to, b, t), pf, dv[b]);
          dk[b] = mfma(rd_tr(qt, to, b, t), sf, dk[b]);
        }
      }
    }
  };

  const int n = nqb_all - qb0;
  if (n > 0) issue(lds0, qb0);
  stage_sync();
  int i = 0;
  for (; i + 1 < n; i += 2) {
    issue(lds1, qb0 + i + 1);
    compute(lds0, qb0 + i);
    stage_sync();
    if (i + 2 < n) issue(lds0, qb0 + i + 2);
    compute(lds1, qb0 + i + 1);
    stage_sync();
  }
  if (i < n) compute(lds0, qb0 + i);
  __syncthreads();  // every wave is done with the tiles: lds0 holds the output rows

  bf16* dK = p.out + (long)zb * p.s * ld + p.h + zh * HD;
  store_rows_lds(dk, lds0 + wave * 32 * ROWB, dK, ld, k0w, p.s, lane, p.scale);
  store_rows_lds(dv, lds0 + wave * 32 * ROWB, dK + p.h, ld, k0w, p.s, lane, 1.0f);
}

// Backward over query blocks: dQ.  Per wave: 32 queries (Q and dO rows
// stationary in registers); key blocks of 64 staged in LDS (K, V).  Per wave
// and key block: S^T = K Q^T, dP^T = V dO^T (lane column = query), P, dS as
// above; dQ^T += K^T dS^T.

// Stationary operands of a wave's 32 queries: Q and dO fragments, this lane's
// query's log-sum-exp and Dv = rowsum(dO o O).  Each half-wave holds half of
// a row (the same columns as its dO fragments); Dv is written for the
// key-block kernel, which runs after this one.
struct BwdQRows {
  bf16x8 qf[HD / 16], of[HD / 16];
  float Lq, Dq;
  __device__ __forceinline__ void load_rows(const AttnArgs& p, int z, int qq, int lane) {
    const int zb = z / p.heads, zh = z % p.heads;
    const long ld = 3L * p.h;
    load_stationary(qf, p.qkv + (long)zb * p.s * ld + zh * HD, ld, qq, p.s, lane);
    load_stationary(of, p.dout + (long)zb * p.s * p.h + zh * HD, p.h, qq, p.s, lane);
  }
  __device__ __forceinline__ void load(const AttnArgs& p, int z, int qq, int lane, bool write_dv) {
    const int zb = z / p.heads, zh = z % p.heads;
    load_rows(p, z, qq, lane);
    Lq = qq < p.s ? p.lse[(long)z * p.s + qq] : 0.f;
    bf16x8 ofr[HD / 16];
    load_stationary(ofr, p.o + (long)zb * p.s * p.h + zh * HD, p.h, qq, p.s, lane);
    float t = 0.f;
#pragma unroll
    for (int ks = 0; ks < HD / 16; ++ks)
#pragma unroll
      for (int e = 0; e < 8; ++e) t += (float)of[ks][e] * (float)ofr[ks][e];
    Dq = t + __shfl_xor(t, 32, 64);
    if (write_dv && lane < 32 && qq < p.s) p.dv[(long)z * p.s + qq] = Dq;
  }
};

// One key block (keys k0..k0+63; K tile kt, V tile vt) for the wave's queries
// q0..q0+31.
template <bool CAUSAL>
__device__ __forceinline__ void bwdq_block(f32x16 (&dq)[HD / 32], const BwdQRows& w, const char* kt,
                                           const char* vt, const RowOffs& ro, const TrOffs& to, int k0,
                                           int q0, int qq, int lane, const AttnArgs& p) {
  if (CAUSAL && k0 > q0 + 31) return;
  const bool need_mask = uniform((CAUSAL && k0 + 63 > q0) || (k0 + 64 > p.s));
  const int room = key_room<CAUSAL>(k0, qq, lane, p);
  // the two 32-key halves of the block in turn (one half's scores live)
#pragma unroll 1
  for (int j = 0; j < 2; ++j) {
    if (CAUSAL && k0 + 32 * j > q0 + 31) break;  // this half is after every query of the wave
    f32x16 sc[1], dp;
    zero(sc[0]);
    zero(dp);
    two_chains<2>(sc[0], kt, j, w.qf, dp, vt, j, w.of, ro);
#pragma unroll
    for (int r = 0; r < 16; ++r) sc[0][r] = __builtin_amdgcn_exp2f(sc[0][r] * p.sl2 - w.Lq);
    if (need_mask) mask_scores<1>(sc, room - 32 * j, 0.f);
#pragma unroll
    for (int r = 0; r < 16; ++r) dp[r] = sc[0][r] * (dp[r] - w.Dq);
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const bf16x8 sf = pack_half(dp, hf);
#pragma unroll
      for (int b = 0; b < HD / 32; ++b) dq[b] = mfma(rd_tr(kt, to, b, 2 * j + hf), sf, dq[b]);
    }
  }
}

// dQ rows q0..q0+31 of the wave (this lane's qq); through LDS area t (8 KB)
// when given.
__device__ __forceinline__ void store_dq(const f32x16 (&dq)[HD / 32], const AttnArgs& p, int z, int q0,
                                         int qq, int lane, char* t = nullptr) {
  const int zb = z / p.heads, zh = z % p.heads;
  const long ld = 3L * p.h;
  bf16* const out = p.out + (long)zb * p.s * ld + zh * HD;
  if (t)
    store_rows_lds(dq, t, out, ld, q0, p.s, lane, p.scale);
  else
    store_dT(dq, out, ld, qq, p.s, lane, p.scale);
}

// One query block of 128 per workgroup (4 waves), two stages of K and V.
template <bool CAUSAL>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_bwd_q_k(AttnArgs p) {
  __shared__ __attribute__((aligned(1024))) char lds0[2 * TILE64];
  __shared__ __attribute__((aligned(1024))) char lds1[2 * TILE64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nqb = (p.s + 127) / 128;
  int z, qb;
  block_of(p, nqb, CAUSAL, z, qb);
  const int zb = z / p.heads, zh = z % p.heads;
  const long ld = 3L * p.h;
  const bf16* Q = p.qkv + (long)zb * p.s * ld + zh * HD;
  const i32x4 rk = make_rsrc(Q + p.h, 2L * p.s * ld);
  const i32x4 rv = make_rsrc(Q + 2 * p.h, 2L * p.s * ld);
  const int q0 = qb * 128 + 32 * wave;
  const int qq = q0 + (lane & 31);

  BwdQRows w;
  w.load(p, z, qq, lane, true);
  RowOffs ro;
  ro.init(lane);
  TrOffs to;
  to.init(lane);

  f32x16 dq[HD / 32];
#pragma unroll
  for (int b = 0; b < HD / 32; ++b) zero(dq[b]);
  const int nkb_all = (p.s + 63) / 64;
  const int nkb = CAUSAL ? min(nkb_all, 2 * qb + 2) : nkb_all;

  auto issue = [&](char* t, int kb) {
    load_tile<64>(rk, t, wave, lane, ld, kb * 64, p.s);
    load_tile<64>(rv, t + TILE64, wave, lane, ld, kb * 64, p.s);
  };
  auto compute = [&](const char* t, int kb) {
    bwdq_block<CAUSAL>(dq, w, t, t + TILE64, ro, to, kb * 64, q0, qq, lane, p);
  };

  if (nkb > 0) issue(lds0, 0);
  stage_sync();
  int kb = 0;
  for (; kb + 1 < nkb; kb += 2) {
    issue(lds1, kb + 1);
    compute(lds0, kb);
    stage_sync();
    if (kb + 2 < nkb) issue(lds0, kb + 2);
    compute(lds1, kb + 1);
    stage_sync();
  }
  if (kb < nkb) compute(lds0, kb);
  __syncthreads();  // every wave is done with the tiles: lds0 holds the output rows
  store_dq(dq, p, z, q0, qq, lane, lds0 + wave * 32 * ROWB);
}

// Causal dQ over pairs of query blocks: the work split of attn_fwd_pair_k
// (waves 0-3: all of qa, then the first key blocks of qb; waves 4-7: the rest
// of qb).  Group 1 forms the log-sum-exp and Dv of qb's rows, writes Dv to
// memory and leaves both in LDS for group 0, which then reloads only the Q
// and dO rows when it moves to qb.  The two partial sums of qb's dQ are added
// through LDS (group 0's first).
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_bwd_q_pair_k(AttnArgs p) {
  __shared__ __attribute__((aligned(1024))) char lds[2 * FWD_GROUP + 3072];
  float2* const stats = (float2*)(lds + 2 * FWD_GROUP);  // qb's (log-sum-exp, Dv) per [wave][lane]
  char* const sink = lds + 2 * FWD_GROUP + 2048;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int grp = wave >> 2, wg = wave & 3;
  const int nqb = (p.s + 127) / 128;
  const int z = blockIdx.x % p.bh, pr = blockIdx.x / p.bh;
  const int qa = pr, qb = nqb - 1 - pr;
  const int nkb_all = (p.s + 63) / 64;
  const int nb = min(nkb_all, 2 * qb + 2);
  const int na = qa == qb ? 0 : min(nkb_all, 2 * qa + 2);
  const int half = (na + nb + 1) / 2;
  const int j0 = grp ? half : 0;
  const int cnt = grp ? na + nb - half : half;
  const int zb = z / p.heads, zh = z % p.heads;
  const long ld = 3L * p.h;
  const bf16* Q = p.qkv + (long)zb * p.s * ld + zh * HD;
  const i32x4 rk = make_rsrc(Q + p.h, 2L * p.s * ld);
  const i32x4 rv = make_rsrc(Q + 2 * p.h, 2L * p.s * ld);
  const i32x4 rq = make_rsrc(Q, 2L * p.s * ld);
  const i32x4 rdo = make_rsrc(p.dout + (long)zb * p.s * p.h + zh * HD, 2L * p.s * p.h);

  int qcur = j0 < na ? qa : qb;
  int q0 = qcur * 128 + 32 * wg;
  int qq = q0 + (lane & 31);
  BwdQRows w;
  w.load(p, z, qq, lane, grp == 1 || qcur != qb);  // group 1 writes qb's Dv, group 0 qa's
  if (grp == 1) stats[wg * 64 + lane] = make_float2(w.Lq, w.Dq);  // read after the first barrier
  RowOffs ro;
  ro.init(lane);
  TrOffs to;
  to.init(lane);
#pragma unroll
  for (int ks = 0; ks < HD / 16; ++ks) ro.off[ks] += grp * FWD_GROUP;
#pragma unroll
  for (int b = 0; b < HD / 32; ++b) {
    to.off[b][0] += grp * FWD_GROUP;
    to.off[b][1] += grp * FWD_GROUP;
  }
  f32x16 dq[HD / 32];
#pragma unroll
  for (int b = 0; b < HD / 32; ++b) zero(dq[b]);

  auto key_block = [&](int j) { return j < na ? j : j - na; };
  auto issue = [&](char* t, int j) {
    char* g = t + grp * FWD_GROUP;
    const int kb = key_block(j);
    load_tile<64>(rk, g, wg, lane, ld, kb * 64, p.s);
    load_tile<64>(rv, g + TILE64, wg, lane, ld, kb * 64, p.s);
  };
  // step it of this group: (on moving to qb, its rows first), the copy of the
  // next step's tiles, then the products
  auto step = [&](int it, const char* cur, char* nxt) {
    const int j = j0 + it;
    if (it < cnt && j == na && qcur != qb) {  // group 0 leaves qa: its rows are complete
      store_dq(dq, p, z, q0, qq, lane);
#pragma unroll
      for (int b = 0; b < HD / 32; ++b) zero(dq[b]);
      qcur = qb;
      q0 = qcur * 128 + 32 * wg;
      qq = q0 + (lane & 31);
      w.load_rows(p, z, qq, lane);
      vm_drain();
      const float2 st2 = stats[wg * 64 + lane];
      w.Lq = st2.x;
      w.Dq = st2.y;
    }
    if (it < cnt && j + 1 == na) {
      warm_rows32(rq, sink, lane, ld, qb * 128 + 32 * wg, p.s);
      warm_rows32(rdo, sink, lane, p.h, qb * 128 + 32 * wg, p.s);
    }
    if (it + 1 < cnt) issue(nxt, j + 1);
    if (it < cnt) bwdq_block<true>(dq, w, cur, cur + TILE64, ro, to, key_block(j) * 64, q0, qq, lane, p);
  };

  if (cnt > 0) issue(lds, j0);
  stage_sync();
  int it = 0;
  for (; it + 1 < half; it += 2) {
    step(it, lds, lds + FWD_STAGE);
    stage_sync();
    step(it + 1, lds + FWD_STAGE, lds);
    stage_sync();
  }
  if (it < half) {
    step(it, lds, lds + FWD_STAGE);
    stage_sync();
  }

  if (grp == 0) {
    if (qcur != qb) {  // no step of qb in this half: qa is complete, qb's share is zero
      store_dq(dq, p, z, q0, qq, lane, lds + FWD_GROUP + 4 * 32 * ROWB + wg * 32 * ROWB);
#pragma unroll
      for (int b = 0; b < HD / 32; ++b) zero(dq[b]);
    }
    float4* dst = (float4*)lds + wg * 16 * 64 + lane;
#pragma unroll
    for (int b = 0; b < HD / 32; ++b)
#pragma unroll
      for (int c = 0; c < 4; ++c)
        dst[(4 * b + c) * 64] = make_float4(dq[b][4 * c], dq[b][4 * c + 1], dq[b][4 * c + 2], dq[b][4 * c + 3]);
  }
  __syncthreads();
  if (grp == 1) {
    const float4* src = (const float4*)lds + wg * 16 * 64 + lane;
#pragma unroll
    for (int b = 0; b < HD / 32; ++b)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const float4 v = src[(4 * b + c) * 64];
        dq[b][4 * c] = v.x + dq[b][4 * c];
        dq[b][4 * c + 1] = v.y + dq[b][4 * c + 1];
        dq[b][4 * c + 2] = v.z + dq[b][4 * c + 2];
        dq[b][4 * c + 3] = v.w + dq[b][4 * c + 3];
      }
    store_dq(dq, p, z, q0, qq, lane, lds + FWD_GROUP + wg * 32 * ROWB);
  }
}

AttnArgs make_args(const void* qkv, int b, int s, int heads, int h) {
  AttnArgs a;
  a.qkv = (const bf16*)qkv;
  a.o = nullptr;
  a.dout = nullptr;
  a.out = nullptr;
  a.lse = nullptr;
  a.dv = nullptr;
  a.s = s;
  a.heads = heads;
  a.bh = b * heads;
  a.h = h;
  a.scale = 1.0f / std::sqrt((float)HD);
  a.sl2 = a.scale * kLog2e;
  return a;
}

// The paired kernels run one equal-length workgroup per CU.  They are used
// when those workgroups fill the CUs of their last round to 90 % or more, or
// when there are so few that every CU holds at most one anyway (a small
// problem); otherwise the per-block kernels, whose uneven blocks the
// hardware packs two to a CU, lose less to the last round.
bool pair_grid_fills(long wgs) {
  const long cus = device_compute_units();
  if (2 * wgs <= cus) return true;
  const long rounds = (wgs + cus - 1) / cus;
  return 10 * wgs >= 9 * rounds * cus;
}

}  // namespace

bool attn_flash_supported(int elt, int head_dim) { return elt == 2 && head_dim == HD; }

bool attn_flash_paired(int b, int s, int heads) {
  const int nqb = (s + 127) / 128;
  return pair_grid_fills((long)((nqb + 1) / 2) * b * heads);
}

hipError_t attn_flash_forward(const void* qkv, void* o, float* lse, int b, int s, int heads, int h,
                              int causal, hipStream_t st) {
  if (h != heads * HD) return hipErrorInvalidValue;
  if (b <= 0 || s <= 0) return hipSuccess;
  AttnArgs a = make_args(qkv, b, s, heads, h);
  a.out = (bf16*)o;
  a.lse = lse;
  const int nqb = (s + 127) / 128;
  const long pairs = (long)((nqb + 1) / 2) * a.bh;
  if (causal && pair_grid_fills(pairs)) {
    hipLaunchKernelGGL(attn_fwd_pair_k, dim3(pairs), dim3(512), 0, st, a);
    return hipGetLastError();
  }
  const dim3 grid(nqb * a.bh);
  if (causal)
    hipLaunchKernelGGL(attn_fwd_k<true>, grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(attn_fwd_k<false>, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t attn_flash_backward(const void* qkv, const void* o, const void* dout, const float* lse,
                               float* dv_scratch, void* dqkv, int b, int s, int heads, int h, int causal,
                               hipStream_t st) {
  if (h != heads * HD) return hipErrorInvalidValue;
  if (b <= 0 || s <= 0) return hipSuccess;
  AttnArgs a = make_args(qkv, b, s, heads, h);
  a.o = (const bf16*)o;
  a.dout = (const bf16*)dout;
  a.out = (bf16*)dqkv;
  a.lse = (float*)lse;
  a.dv = dv_scratch;
  // the query-block kernel also writes Dv, which the key-block kernel reads
  const int nqb = (s + 127) / 128;
  const long pairs = (long)((nqb + 1) / 2) * a.bh;
  const dim3 grid(nqb * a.bh);
  if (causal) {
    if (pair_grid_fills(pairs))
      hipLaunchKernelGGL(attn_bwd_q_pair_k, dim3(pairs), dim3(512), 0, st, a);
    else
      hipLaunchKernelGGL(attn_bwd_q_k<true>, grid, dim3(256), 0, st, a);
    hipLaunchKernelGGL(attn_bwd_kv_k<true>, grid, dim3(256), 0, st, a);
  } else {
    hipLaunchKernelGGL(attn_bwd_q_k<false>, grid, dim3(256), 0, st, a);
    hipLaunchKernelGGL(attn_bwd_kv_k<false>, grid, dim3(256), 0, st, a);
  }
  return hipGetLastError();
}
