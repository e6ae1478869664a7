// Stage runtime behind the C ABI of include/recycle_stage.h.
//
// One handle = pipeline stage i on data-parallel pipeline k_s.  It owns no
// device memory: three caller arenas hold
//   state: flat fp32 master weights | fp32 gradients | Adam m | Adam v, then
//          the bf16 copies of the weight matrices (bf16 stages).  Matrices of
//          all layers come first, so weight decay applies to one prefix.
//   stash: the WeightGradStore (ReCycle, section 5): max_stashed_mb weight-pass
//          slots (held from F to W) and max_inflight_mb forward-only slots
//          (held from F to B), each laid out per layer.
//   work:  scratch reused by every call (attention scores, dO, reduction partials).
// Each call checks the micro-batch state machine on the host first, then
// enqueues its kernel sequence on the handle's stream and returns.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <cmath>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "gemm.h"
#include "kernels.h"
#include "recycle_stage.h"

namespace {

thread_local std::string g_err;

rc_status fail(rc_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

#define HIPCHK(expr)                                                                     \
  do {                                                                                   \
    hipError_t e_ = (expr);                                                              \
    if (e_ != hipSuccess)                                                                \
      return fail(RC_ERR_HIP, std::string(#expr) + ": " + hipGetErrorString(e_));        \
  } while (0)

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
long pad64(long n) { return (n + 63) / 64 * 64; }

const int kMatrixIds[4] = {RC_P_W_QKV, RC_P_W_O, RC_P_W_1, RC_P_W_2};
const int kVectorIds[8] = {RC_P_LN1_G, RC_P_LN1_B, RC_P_B_QKV, RC_P_B_O,
                           RC_P_LN2_G, RC_P_LN2_B, RC_P_B_1, RC_P_B_2};

struct PLoc {
  long off = 0, count = 0;
};

// Byte offsets inside one layer of a weight-pass slot.
struct WLayer {
  size_t X, A, O, H, C, G, dY, dQKV, dH, dU, dA, dC, mu1, r1, mu2, r2, bytes;
};
// Byte offsets inside one layer of a forward-only slot.
struct FLayer {
  // Dg: gelu'(U) of the FFN, which the FC2 input gradient multiplies by (the
  // forward stores it instead of U: the same information for B_input, and the
  // derivative is formed where the fp32 U is at hand).  P: attention
  // probabilities, or the row log-sum-exp (fused attention).
  size_t QKV, Dg, P, bytes;
};

struct Layout {
  int L, h, a, d, f, s, b, elt, causal;
  long T;
  bool bf, flash;
  float eps;
  int wslots, fslots;
  std::vector<std::array<PLoc, RC_NUM_PARAMS>> p;
  long n_mat, n_total;
  size_t off_master, off_grad, off_m, off_v, off_wb, state_bytes;
  WLayer w;
  FLayer fl;
  size_t wslot_bytes, fslot_bytes, off_fslots, stash_bytes;
  size_t off_S, off_dS, off_dO, off_dv, off_check, off_part, off_cswork, work_bytes;
  uint64_t acct_af, acct_sw;
};

rc_status make_layout(const rc_stage_config* c, Layout& y) {
  if (!c) return fail(RC_ERR_INVALID_ARG, "null config");
  if (c->num_layers < 1 || c->hidden < 1 || c->heads < 1 || c->ffn < 1 || c->seq_len < 1 ||
      c->micro_batch < 1)
    return fail(RC_ERR_INVALID_ARG, "config sizes must be positive");
  if (c->dtype != RC_FP32 && c->dtype != RC_BF16) return fail(RC_ERR_INVALID_ARG, "unknown dtype");
  if (c->causal != 0 && c->causal != 1) return fail(RC_ERR_INVALID_ARG, "causal must be 0 or 1");
  if (c->max_stashed_mb < 1 || c->max_inflight_mb < 1 || c->max_inflight_mb > c->max_stashed_mb)
    return fail(RC_ERR_INVALID_ARG, "need 1 <= max_inflight_mb <= max_stashed_mb");
  if (!(c->ln_eps >= 0.f)) return fail(RC_ERR_INVALID_ARG, "ln_eps must be >= 0");
  if (c->hidden % c->heads) return fail(RC_ERR_UNSUPPORTED, "hidden must be a multiple of heads");
  const int d = c->hidden / c->heads;
  if (c->hidden % 8 || c->ffn % 8 || c->seq_len % 8 || d % 8)
    return fail(RC_ERR_UNSUPPORTED, "hidden, ffn, seq_len and head_dim must be multiples of 8");
  if (c->dtype == RC_BF16) {
    // The matrix-core kernels address their operands through buffer
    // descriptors whose range is 2^31 - 1 bytes (beyond it a load returns
    // zeros), so every matrix they read must fit one.
    const long cap = 0x7fffffffL, wide = std::max(3L * c->hidden, (long)c->ffn);
    const long T = (long)c->micro_batch * c->seq_len;
    if (2 * T * wide > cap)
      return fail(RC_ERR_UNSUPPORTED, "bf16 activation matrix [micro_batch*seq_len, max(3*hidden, ffn)] "
                                      "exceeds 2^31-1 bytes");
    if (2L * c->hidden * wide > cap)
      return fail(RC_ERR_UNSUPPORTED, "bf16 weight matrix [hidden, max(3*hidden, ffn)] exceeds 2^31-1 bytes");
    if (!attn_flash_supported(2, d) && 2L * c->seq_len * c->seq_len > cap)
      return fail(RC_ERR_UNSUPPORTED, "bf16 attention probabilities [seq_len, seq_len] of one head "
                                      "exceed 2^31-1 bytes");
  }
  y.L = c->num_layers;
  y.h = c->hidden;
  y.a = c->heads;
  y.d = d;
  y.f = c->ffn;
  y.s = c->seq_len;
  y.b = c->micro_batch;
  y.T = (long)c->micro_batch * c->seq_len;
  y.bf = c->dtype == RC_BF16;
  y.elt = y.bf ? 2 : 4;
  y.flash = attn_flash_supported(y.elt, d);
  y.causal = c->causal;
  y.eps = c->ln_eps;
  y.wslots = c->max_stashed_mb;
  y.fslots = c->max_inflight_mb;
  const long h = y.h, f = y.f;
  const long msize[RC_NUM_PARAMS] = {h, h, h * 3 * h, 3 * h, h * h, h, h, h, h * f, f, f * h, h};
  y.p.assign(y.L, {});
  long off = 0;
  for (int l = 0; l < y.L; ++l)
    for (int pid : kMatrixIds) {
      y.p[l][pid] = {off, msize[pid]};
      off += pad64(msize[pid]);
    }
  y.n_mat = off;
  for (int l = 0; l < y.L; ++l)
    for (int pid : kVectorIds) {
      y.p[l][pid] = {off, msize[pid]};
      off += pad64(msize[pid]);
    }
  y.n_total = off;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t r = o;
    o = align_up(o + bytes);
    return r;
  };
  y.off_master = take(4 * y.n_total);
  y.off_grad = take(4 * y.n_total);
  y.off_m = take(4 * y.n_total);
  y.off_v = take(4 * y.n_total);
  y.off_wb = take(y.bf ? 2 * y.n_mat : 0);
  y.state_bytes = o;

  const size_t E = y.elt, T = y.T;
  o = 0;
  WLayer& w = y.w;
  w.X = take(T * h * E);
  w.A = take(T * h * E);
  w.O = take(T * h * E);
  w.H = take(T * h * E);
  w.C = take(T * h * E);
  w.G = take(T * f * E);
  w.dY = take(T * h * E);
  w.dQKV = take(T * 3 * h * E);
  w.dH = take(T * h * E);
  w.dU = take(T * f * E);
  w.dA = take(T * h * E);
  w.dC = take(T * h * E);
  w.mu1 = take(T * 4);
  w.r1 = take(T * 4);
  w.mu2 = take(T * 4);
  w.r2 = take(T * 4);
  w.bytes = o;
  o = 0;
  const size_t ss = (size_t)y.b * y.a * y.s * y.s;
  const size_t rows = (size_t)y.b * y.a * y.s;
  y.fl.QKV = take(T * 3 * h * E);
  y.fl.Dg = take(T * f * E);
  y.fl.P = take(y.flash ? rows * 4 : ss * E);
  y.fl.bytes = o;
  y.wslot_bytes = (size_t)y.L * w.bytes;
  y.fslot_bytes = (size_t)y.L * y.fl.bytes;
  y.off_fslots = (size_t)y.wslots * y.wslot_bytes;
  y.stash_bytes = y.off_fslots + (size_t)y.fslots * y.fslot_bytes;
  o = 0;
  y.off_S = take(y.flash ? 0 : ss * 4);
  y.off_dS = take(y.flash ? 0 : ss * E);
  y.off_dO = take(T * h * E);
  y.off_dv = take(y.flash ? rows * 4 : 0);
  y.off_check = take(8 * GRAD_CHECK_BLOCKS);
  // Logical stash bytes per micro-batch (tensor sizes, no alignment padding):
  // from F to B_input the forward-written part of the weight-pass slot (X, A,
  // O, H, C, G and the LayerNorm statistics) plus the forward-only slot (QKV,
  // gelu'(U) and the attention row statistics or probabilities); from B_input to
  // B_weight the whole weight-pass slot.
  {
    const uint64_t Th = (uint64_t)T * h, Tf = (uint64_t)T * f, st = 16ull * T;
    const uint64_t attn = y.flash ? 4ull * rows : (uint64_t)E * ss;
    y.acct_af = (uint64_t)y.L * (E * (8 * Th + 2 * Tf) + st + attn);
    y.acct_sw = (uint64_t)y.L * (E * (12 * Th + 2 * Tf) + st);
  }
  y.off_part = take(4 * colsum_part_floats(y.T, (int)std::max(3 * h, f),
                                           std::min(y.wslots, (int)GEMM_MAX_SEG)));
  // partial bias sums of the bf16 weight-gradient products (one product at a
  // time): the largest of [h, 3h], [h, h], [h, f], [f, h]
  y.off_cswork = take(y.bf ? 4 * std::max(gemm_colsum_floats(h, std::max(3 * h, f)), gemm_colsum_floats(f, h))
                           : 0);
  y.work_bytes = o;
  return RC_OK;
}

struct MbRec {
  int state;  // 1 = F done, 2 = B done, 3 = W done
  int ws, fs;
};

}  // namespace

struct rc_stage {
  rc_stage_config cfg;
  rc_adam_config adam;
  int stage_index, pipeline_id;
  bool dry;
  hipStream_t stream;
  char *state, *stash, *work;
  Layout lay;
  std::map<std::pair<int, int>, MbRec> mbs;
  std::vector<int> free_w, free_f;
  std::vector<rc_op_record> log;
  int64_t iter = 0, t = 0;
  bool grads_fresh = true;
  // Post-step validation: `closed` = the last call closed an iteration (step,
  // skip, rollback); a step can be rolled back while it is the last call.
  bool closed = false, can_rollback = false;
  float last_scale = 1.f;
  // Stash accounting: bytes held by micro-batches between calls, its maximum,
  // and the limit a forward pass must respect (0: none).
  uint64_t live = 0, peak = 0, limit = 0;
  // per-kernel profile
  struct Rec {
    int kind;
    hipEvent_t a, b;
    double flops, bytes;
  };
  bool prof = false;
  std::vector<Rec> pending;
  std::vector<hipEvent_t> pool;
  rc_kernel_stat stats[RC_K_COUNT];
};

namespace {

struct WPtr {
  char *X, *A, *O, *H, *C, *G, *dY, *dQKV, *dH, *dU, *dA, *dC;
  float *mu1, *r1, *mu2, *r2;
};
struct FPtr {
  char *QKV, *Dg, *P;
};

WPtr wptr(rc_stage* st, int slot, int l) {
  const Layout& y = st->lay;
  char* b = st->stash + (size_t)slot * y.wslot_bytes + (size_t)l * y.w.bytes;
  const WLayer& w = y.w;
  return {b + w.X, b + w.A, b + w.O, b + w.H, b + w.C, b + w.G, b + w.dY, b + w.dQKV,
          b + w.dH, b + w.dU, b + w.dA, b + w.dC, (float*)(b + w.mu1), (float*)(b + w.r1),
          (float*)(b + w.mu2), (float*)(b + w.r2)};
}

FPtr fptr(rc_stage* st, int slot, int l) {
  const Layout& y = st->lay;
  char* b = st->stash + y.off_fslots + (size_t)slot * y.fslot_bytes + (size_t)l * y.fl.bytes;
  return {b + y.fl.QKV, b + y.fl.Dg, b + y.fl.P};
}

float* master(rc_stage* st, int l, int pid) {
  return (float*)(st->state + st->lay.off_master) + st->lay.p[l][pid].off;
}
float* gradp(rc_stage* st, int l, int pid) {
  return (float*)(st->state + st->lay.off_grad) + st->lay.p[l][pid].off;
}
// Weight matrix as read by the GEMMs: the bf16 copy for bf16 stages.
const void* weight(rc_stage* st, int l, int pid) {
  if (st->lay.bf) return (const char*)(st->state + st->lay.off_wb) + 2 * st->lay.p[l][pid].off;
  return master(st, l, pid);
}

// Element offset into an activation buffer.
inline char* el(void* p, long n, int elt) { return (char*)p + n * elt; }

// Records a HIP event pair around the enclosed launches when profiling.
struct Prof {
  rc_stage* st;
  int kind;
  double flops, bytes;
  hipEvent_t a = nullptr;
  Prof(rc_stage* s, int k, double fl, double by) : st(s), kind(k), flops(fl), bytes(by) {
    if (st->prof) a = next_event(st);
  }
  ~Prof() {
    if (!st->prof || !a) return;
    hipEvent_t b = next_event(st);
    if (b) st->pending.push_back({kind, a, b, flops, bytes});
  }
  static hipEvent_t next_event(rc_stage* st) {
    hipEvent_t e = nullptr;
    if (!st->pool.empty()) {
      e = st->pool.back();
      st->pool.pop_back();
    } else if (hipEventCreate(&e) != hipSuccess) {
      return nullptr;
    }
    hipEventRecord(e, st->stream);
    return e;
  }
};

double gemm_bytes(long M, long N, long K, int in_elt, int out_bytes) {
  return (double)in_elt * ((double)M * K + (double)K * N) + (double)out_bytes * M * N;
}

GemmParams gp(int M, int N, int K, const void* A, long lda, int ak, const void* B, long ldb, int bk,
              int epi, void* C, long ldc) {
  GemmParams g;
  std::memset(&g, 0, sizeof(g));
  g.M = M;
  g.N = N;
  g.K = K;
  g.A = A;
  g.lda = lda;
  g.a_kcontig = ak;
  g.B = B;
  g.ldb = ldb;
  g.b_kcontig = bk;
  g.batch = 1;
  g.heads = 1;
  g.epi = epi;
  g.C = C;
  g.ldc = ldc;
  return g;
}

hipError_t gemm(rc_stage* st, const GemmParams& g) {
  return st->lay.bf ? gemm_bf16(g, st->stream) : gemm_f32(g, st->stream);
}

// A linear-layer GEMM, profiled as one launch of class `kind`.
hipError_t gemm_lin(rc_stage* st, const GemmParams& g, int kind) {
  const int E = st->lay.elt;
  int ob = E;
  if (g.epi == EPI_F32_ACC) ob = g.accumulate ? 8 : 4;
  if (g.epi == EPI_BIAS_GELU) ob = 2 * E;
  if (g.epi == EPI_BIAS_RESID || g.epi == EPI_GELU_BWD) ob = 2 * E;
  Prof pr(st, kind, 2.0 * g.M * (double)g.N * g.K, gemm_bytes(g.M, g.N, g.K, E, ob));
  return gemm(st, g);
}

// Per (sequence, head) batching of the attention products; Q, K, V and dQ,
// dK, dV live as column blocks of the [T, 3h] QKV / dQKV matrices and O, dO
// as head columns of [T, h] matrices.
void batch_heads(GemmParams& g, const Layout& y, long a_bs, long a_hs, long b_bs, long b_hs,
                 long c_bs, long c_hs) {
  g.batch = y.b;
  g.heads = y.a;
  g.a_bs = a_bs;
  g.a_hs = a_hs;
  g.b_bs = b_bs;
  g.b_hs = b_hs;
  g.c_bs = c_bs;
  g.c_hs = c_hs;
}

rc_status attn_forward(rc_stage* st, char* QKV, char* P, char* O) {
  const Layout& y = st->lay;
  const int E = y.elt;
  if (y.flash) {
    HIPCHK(attn_flash_forward(QKV, O, (float*)P, y.b, y.s, y.a, y.h, y.causal, st->stream));
    return RC_OK;
  }
  const long s = y.s, h = y.h, d = y.d, ss = s * s;
  float* S = (float*)(st->work + y.off_S);
  GemmParams g = gp(y.s, y.s, y.d, QKV, 3 * h, 1, el(QKV, h, E), 3 * h, 1, EPI_F32_STORE, S, s);
  batch_heads(g, y, s * 3 * h, d, s * 3 * h, d, y.a * ss, ss);
  g.causal_skip = y.causal;
  HIPCHK(gemm(st, g));
  HIPCHK(softmax_forward(E, S, P, (long)y.b * y.a * y.s, y.s, 1.0f / std::sqrt((float)y.d),
                         y.causal, st->stream));
  g = gp(y.s, y.d, y.s, P, s, 1, el(QKV, 2 * h, E), 3 * h, 0, EPI_STORE, O, h);
  batch_heads(g, y, y.a * ss, ss, s * 3 * h, d, s * h, d);
  g.krange = y.causal ? KR_BELOW : KR_FULL;
  HIPCHK(gemm(st, g));
  return RC_OK;
}

rc_status attn_backward(rc_stage* st, char* QKV, char* P, char* O, char* dO, char* dQKV) {
  const Layout& y = st->lay;
  const int E = y.elt;
  if (y.flash) {
    HIPCHK(attn_flash_backward(QKV, O, dO, (const float*)P, (float*)(st->work + y.off_dv), dQKV, y.b,
                               y.s, y.a, y.h, y.causal, st->stream));
    return RC_OK;
  }
  const long s = y.s, h = y.h, d = y.d, ss = s * s;
  float* dP = (float*)(st->work + y.off_S);
  char* dS = st->work + y.off_dS;
  GemmParams g = gp(y.s, y.s, y.d, dO, h, 1, el(QKV, 2 * h, E), 3 * h, 1, EPI_F32_STORE, dP, s);
  batch_heads(g, y, s * h, d, s * 3 * h, d, y.a * ss, ss);
  g.causal_skip = y.causal;
  HIPCHK(gemm(st, g));
  HIPCHK(softmax_backward(E, dP, P, dS, (long)y.b * y.a * y.s, y.s, 1.0f / std::sqrt((float)y.d),
                          y.causal, st->stream));
  // dQ = dS K
  g = gp(y.s, y.d, y.s, dS, s, 1, el(QKV, h, E), 3 * h, 0, EPI_STORE, dQKV, 3 * h);
  batch_heads(g, y, y.a * ss, ss, s * 3 * h, d, s * 3 * h, d);
  g.krange = y.causal ? KR_BELOW : KR_FULL;
  HIPCHK(gemm(st, g));
  // dK = dS^T Q
  g = gp(y.s, y.d, y.s, dS, s, 0, QKV, 3 * h, 0, EPI_STORE, el(dQKV, h, E), 3 * h);
  batch_heads(g, y, y.a * ss, ss, s * 3 * h, d, s * 3 * h, d);
  g.krange = y.causal ? KR_ABOVE : KR_FULL;
  HIPCHK(gemm(st, g));
  // dV = P^T dO
  g = gp(y.s, y.d, y.s, P, s, 0, dO, h, 0, EPI_STORE, el(dQKV, 2 * h, E), 3 * h);
  batch_heads(g, y, y.a * ss, ss, s * h, d, s * 3 * h, d);
  g.krange = y.causal ? KR_ABOVE : KR_FULL;
  HIPCHK(gemm(st, g));
  return RC_OK;
}

rc_status run_forward(rc_stage* st, int ws, int fs, const void* x, void* yout) {
  const Layout& y = st->lay;
  const int E = y.elt, L = y.L;
  const long T = y.T, h = y.h, f = y.f;
  hipStream_t s = st->stream;
  const double ln_f_bytes = 2.0 * T * h * E + 8.0 * T + 8.0 * h;
  const double att = (y.causal ? 1.0 : 2.0) * y.b * (double)y.s * y.s * h;
  for (int l = 0; l < L; ++l) {
    WPtr w = wptr(st, ws, l);
    FPtr fl = fptr(st, fs, l);
    {
      // layer 0 reads the caller's x and also copies it into the stash
      Prof pr1(st, RC_K_LN, 0, ln_f_bytes + (l == 0 ? (double)T * h * E : 0.0));
      HIPCHK(ln_forward(E, l == 0 ? x : w.X, master(st, l, RC_P_LN1_G), master(st, l, RC_P_LN1_B), w.A,
                        w.mu1, w.r1, T, y.h, y.eps, s, l == 0 ? w.X : nullptr));
    }
    GemmParams g = gp(T, 3 * h, h, w.A, h, 1, weight(st, l, RC_P_W_QKV), 3 * h, 0, EPI_BIAS, fl.QKV, 3 * h);
    g.bias = master(st, l, RC_P_B_QKV);
    HIPCHK(gemm_lin(st, g, RC_K_GEMM_FWD));
    {
      Prof pa(st, RC_K_ATTN_FWD, 2.0 * att, 4.0 * T * h * E);
      rc_status r = attn_forward(st, fl.QKV, fl.P, w.O);
      if (r != RC_OK) return r;
    }
    g = gp(T, h, h, w.O, h, 1, weight(st, l, RC_P_W_O), h, 0, EPI_BIAS_RESID, w.H, h);
    g.bias = master(st, l, RC_P_B_O);
    g.resid = w.X;
    g.ld_resid = h;
    HIPCHK(gemm_lin(st, g, RC_K_GEMM_FWD));
    {
      Prof pr2(st, RC_K_LN, 0, ln_f_bytes);
      HIPCHK(ln_forward(E, w.H, master(st, l, RC_P_LN2_G), master(st, l, RC_P_LN2_B), w.C, w.mu2,
                        w.r2, T, y.h, y.eps, s));
    }
    g = gp(T, f, h, w.C, h, 1, weight(st, l, RC_P_W_1), f, 0, EPI_BIAS_GELU, fl.Dg, f);
    g.bias = master(st, l, RC_P_B_1);
    g.C2 = w.G;
    g.ldc2 = f;
    HIPCHK(gemm_lin(st, g, RC_K_GEMM_FWD));
    void* out = (l + 1 < L) ? (void*)wptr(st, ws, l + 1).X : yout;
    g = gp(T, h, f, w.G, f, 1, weight(st, l, RC_P_W_2), h, 0, EPI_BIAS_RESID, out, h);
    g.bias = master(st, l, RC_P_B_2);
    g.resid = w.H;
    g.ld_resid = h;
    HIPCHK(gemm_lin(st, g, RC_K_GEMM_FWD));
  }
  return RC_OK;
}

rc_status run_backward_input(rc_stage* st, int ws, int fs, const void* dy, void* dx) {
  const Layout& y = st->lay;
  const int E = y.elt, L = y.L;
  const long T = y.T, h = y.h, f = y.f;
  hipStream_t s = st->stream;
  char* dO = st->work + y.off_dO;
  const double ln_b_bytes = 4.0 * T * h * E + 8.0 * T + 4.0 * h;
  const double att = (y.causal ? 1.0 : 2.0) * y.b * (double)y.s * y.s * h;
  for (int l = L - 1; l >= 0; --l) {
    WPtr w = wptr(st, ws, l);
    FPtr fl = fptr(st, fs, l);
    // The last layer reads the caller's dy; its LN2 backward, which adds dy as
    // the residual, also copies it into the stash for the weight pass.
    const bool top = l == L - 1;
    char* const dYl = top ? (char*)dy : w.dY;
    // dU = (dY W_2^T) * gelu'(U), the derivative stored by the forward
    GemmParams g = gp(T, f, h, dYl, h, 1, weight(st, l, RC_P_W_2), h, 1, EPI_GELU_BWD, w.dU, f);
    g.aux = fl.Dg;
    g.ld_aux = f;
    HIPCHK(gemm_lin(st, g, RC_K_GEMM_DGRAD));
    // dC = dU W_1^T
    g = gp(T, h, f, w.dU, f, 1, weight(st, l, RC_P_W_1), f, 1, EPI_STORE, w.dC, h);
    HIPCHK(gemm_lin(st, g, RC_K_GEMM_DGRAD));
    // dH = dY + LN2^T(dC)
    {
      Prof pr(st, RC_K_LN, 0, ln_b_bytes + (top ? (double)T * h * E : 0.0));
      HIPCHK(ln_backward(E, w.dC, w.H, w.mu2, w.r2, master(st, l, RC_P_LN2_G), dYl, w.dH, T, y.h, s,
                         top ? w.dY : nullptr));
    }
    // dO = dH W_o^T
    g = gp(T, h, h, w.dH, h, 1, weight(st, l, RC_P_W_O), h, 1, EPI_STORE, dO, h);
    HIPCHK(gemm_lin(st, g, RC_K_GEMM_DGRAD));
    {
      Prof pa(st, RC_K_ATTN_BWD, 4.0 * att, 8.0 * T * h * E);
      rc_status r = attn_backward(st, fl.QKV, fl.P, w.O, dO, w.dQKV);
      if (r != RC_OK) return r;
    }
    // dA = dQKV W_qkv^T
    g = gp(T, h, 3 * h, w.dQKV, 3 * h, 1, weight(st, l, RC_P_W_QKV), 3 * h, 1, EPI_STORE, w.dA, h);
    HIPCHK(gemm_lin(st, g, RC_K_GEMM_DGRAD));
    // dX = dH + LN1^T(dA)
    void* out = l > 0 ? (void*)wptr(st, ws, l - 1).dY : dx;
    Prof pr(st, RC_K_LN, 0, ln_b_bytes);
    HIPCHK(ln_backward(E, w.dA, w.X, w.mu1, w.r1, master(st, l, RC_P_LN1_G), w.dH, out, T, y.h, s));
  }
  return RC_OK;
}

// B_weight of n micro-batches (stash slots ws[0..n)) in one pass: every
// parameter's gradient contribution of all n is one product / reduction over
// their concatenated tokens (segments of T tokens, one per stash slot).
rc_status run_backward_weight(rc_stage* st, const int* ws, int n) {
  const Layout& y = st->lay;
  const int E = y.elt;
  const long T = y.T, h = y.h, f = y.f;
  const int acc = st->grads_fresh ? 0 : 1;
  hipStream_t s = st->stream;
  float* part = (float*)(st->work + y.off_part);
  // bf16 k-tiles of 64 must not straddle two micro-batches
  const bool fused = !y.bf || (T % 64 == 0);
  for (int l = 0; l < y.L; ++l) {
    WPtr w[GEMM_MAX_SEG];
    for (int q = 0; q < n; ++q) w[q] = wptr(st, ws[q], l);
    // pid: the weight; bpid: the bias of the same linear layer, whose gradient
    // sum_t dY[t, :] the bf16 weight-gradient product computes on the side
    // from the dY tiles it stages (the fp32 path leaves it to the column sums).
    struct {
      int pid, bpid;
      long M, N;
      char* WPtr::*X;
      char* WPtr::*dY;
    } lin[4] = {{RC_P_W_QKV, RC_P_B_QKV, h, 3 * h, &WPtr::A, &WPtr::dQKV},
                {RC_P_W_O, RC_P_B_O, h, h, &WPtr::O, &WPtr::dH},
                {RC_P_W_1, RC_P_B_1, h, f, &WPtr::C, &WPtr::dU},
                {RC_P_W_2, RC_P_B_2, f, h, &WPtr::G, &WPtr::dY}};
    for (auto& q : lin) {
      // dW (+)= sum over the n micro-batches of X^T dY (reduction over tokens)
      if (fused) {
        GemmParams g = gp(q.M, q.N, T * n, nullptr, q.M, 0, nullptr, q.N, 0, EPI_F32_ACC,
                          gradp(st, l, q.pid), q.N);
        g.accumulate = acc;
        if (y.bf) {
          g.colsum_out = gradp(st, l, q.bpid);
          g.colsum_acc = acc;
          g.colsum_work = (float*)(st->work + y.off_cswork);
        }
        g.kseg_len = (int)T;
        for (int k = 0; k < n; ++k) {
          g.segA[k] = w[k].*(q.X);
          g.segB[k] = w[k].*(q.dY);
        }
        HIPCHK(gemm_lin(st, g, RC_K_GEMM_WGRAD));
      } else {
        for (int k = 0; k < n; ++k) {
          GemmParams g = gp(q.M, q.N, T, w[k].*(q.X), q.M, 0, w[k].*(q.dY), q.N, 0, EPI_F32_ACC,
                            gradp(st, l, q.pid), q.N);
          g.accumulate = acc || k > 0;
          if (y.bf) {
            g.colsum_out = gradp(st, l, q.bpid);
            g.colsum_acc = g.accumulate;
            g.colsum_work = (float*)(st->work + y.off_cswork);
          }
          HIPCHK(gemm_lin(st, g, RC_K_GEMM_WGRAD));
        }
      }
    }
    // Column sums: the LN parameters' gradients, and on the fp32 path also the
    // biases' (bytes: n micro-batches' inputs, then the gradient update).
    const double rb = acc ? 8.0 : 4.0;
    const double bias_in = y.bf ? 0.0 : (double)T * (6 * h + f) * E;
    Prof pr(st, RC_K_REDUCE, 0,
            n * (bias_in + 4.0 * T * h * E + 16.0 * T) + (y.bf ? 0.0 : rb * (6 * h + f)) + 4 * rb * h);
    ColSegs sg;
    std::memset(&sg, 0, sizeof(sg));
    struct {
      int pid;
      long N;
      char* WPtr::*D;
    } bias[4] = {{RC_P_B_QKV, 3 * h, &WPtr::dQKV}, {RC_P_B_O, h, &WPtr::dH},
                 {RC_P_B_1, f, &WPtr::dU}, {RC_P_B_2, h, &WPtr::dY}};
    if (!y.bf) {
      for (auto& b : bias) {
        for (int k = 0; k < n; ++k) sg.dout[k] = w[k].*(b.D);
        HIPCHK(colsum(E, false, sg, n, b.N, T, (int)b.N, nullptr, gradp(st, l, b.pid), acc, part, s));
      }
    }
    for (int k = 0; k < n; ++k) {
      sg.dout[k] = w[k].dA;
      sg.x[k] = w[k].X;
      sg.mean[k] = w[k].mu1;
      sg.rstd[k] = w[k].r1;
    }
    HIPCHK(colsum(E, true, sg, n, h, T, (int)h, gradp(st, l, RC_P_LN1_G), gradp(st, l, RC_P_LN1_B), acc,
                  part, s));
    for (int k = 0; k < n; ++k) {
      sg.dout[k] = w[k].dC;
      sg.x[k] = w[k].H;
      sg.mean[k] = w[k].mu2;
      sg.rstd[k] = w[k].r2;
    }
    HIPCHK(colsum(E, true, sg, n, h, T, (int)h, gradp(st, l, RC_P_LN2_G), gradp(st, l, RC_P_LN2_B), acc,
                  part, s));
  }
  return RC_OK;
}

rc_status run_optimizer(rc_stage* st, float grad_scale) {
  const Layout& y = st->lay;
  hipStream_t s = st->stream;
  float* P = (float*)(st->state + y.off_master);
  float* G = (float*)(st->state + y.off_grad);
  float* M = (float*)(st->state + y.off_m);
  float* V = (float*)(st->state + y.off_v);
  if (st->grads_fresh) HIPCHK(fill_f32(G, y.n_total, 0.f, s));
  const double t = (double)(st->t + 1);
  const rc_adam_config& a = st->adam;
  const double bc1 = 1.0 - std::pow((double)a.beta1, t);
  const double bc2 = 1.0 - std::pow((double)a.beta2, t);
  Prof pr(st, RC_K_ADAM, 0, 28.0 * y.n_total + (y.bf ? 2.0 * y.n_mat : 0.0));
  HIPCHK(adamw_step(P, G, M, V, y.bf ? (void*)(st->state + y.off_wb) : nullptr, y.n_total, y.n_mat,
                    a.lr, a.beta1, a.beta2, a.eps, a.weight_decay, (float)(a.lr / bc1),
                    (float)(1.0 / std::sqrt(bc2)), grad_scale, s));
  return RC_OK;
}

// Undo the step number st->t with the gradients it used (still in the
// gradient buffer: the next iteration's first weight pass overwrites them).
rc_status run_rollback(rc_stage* st) {
  const Layout& y = st->lay;
  const double t = (double)st->t;
  const rc_adam_config& a = st->adam;
  const double bc1 = 1.0 - std::pow((double)a.beta1, t);
  const double bc2 = 1.0 - std::pow((double)a.beta2, t);
  Prof pr(st, RC_K_ADAM, 0, 28.0 * y.n_total + (y.bf ? 2.0 * y.n_mat : 0.0));
  HIPCHK(adamw_undo((float*)(st->state + y.off_master), (const float*)(st->state + y.off_grad),
                    (float*)(st->state + y.off_m), (float*)(st->state + y.off_v),
                    y.bf ? (void*)(st->state + y.off_wb) : nullptr, y.n_total, y.n_mat, a.lr, a.beta1,
                    a.beta2, a.eps, a.weight_decay, (float)(a.lr / bc1), (float)(1.0 / std::sqrt(bc2)),
                    st->last_scale, st->t == 1 ? 1 : 0, st->stream));
  return RC_OK;
}

void record(rc_stage* st, int op, int j, int k) {
  rc_op_record r;
  r.seq = (int64_t)st->log.size();
  r.op = op;
  r.j = j;
  r.k = k;
  r.k_s = st->pipeline_id;
  r.stage = st->stage_index;
  r.reserved = 0;
  r.iter = st->iter;
  st->log.push_back(r);
}

int take_min(std::vector<int>& v) {
  auto it = std::min_element(v.begin(), v.end());
  int x = *it;
  v.erase(it);
  return x;
}

rc_status check_param(rc_stage* st, int layer, int pid) {
  if (!st) return fail(RC_ERR_INVALID_ARG, "null stage");
  if (layer < 0 || layer >= st->lay.L) return fail(RC_ERR_INVALID_ARG, "layer out of range");
  if (pid < 0 || pid >= RC_NUM_PARAMS) return fail(RC_ERR_INVALID_ARG, "param_id out of range");
  if (st->dry) return fail(RC_ERR_INVALID_ARG, "dry-run handle has no device memory");
  return RC_OK;
}

// Work memory of handles made by rc_stage_create_static: one file-scope
// device array, which every GPU the library runs on holds until the process
// ends.  In host code `scratch` names a host-side stand-in, so its device
// address is looked up once per device (hipGetSymbolAddress, with that
// device current) and only that address is handed to kernels.
constexpr size_t kScratchBytes = (size_t)RC_STATIC_WORK_BYTES;
static __device__ __align__(256) char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the device that runs `stream` (the null
// stream: the current device).
rc_status scratch_address(hipStream_t stream, void** out) {
  int cur = 0;
  HIPCHK(hipGetDevice(&cur));
  const int dev = stream ? hipGetStreamDeviceId(stream) : cur;
  if (dev < 0 || dev >= kMaxDevices)
    return fail(RC_ERR_UNSUPPORTED, "no-allocation work memory: device index " + std::to_string(dev) +
                                        " outside 0.." + std::to_string(kMaxDevices - 1));
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    if (dev != cur) HIPCHK(hipSetDevice(dev));
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur) HIPCHK(hipSetDevice(cur));
    if (e != hipSuccess || !p)
      return fail(RC_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return RC_OK;
}

// Shared by rc_stage_create and rc_stage_create_static once the arenas are known.
rc_status create_handle(const Layout& y, const rc_stage_config* cfg, const rc_adam_config* adam,
                        int32_t stage_index, int32_t pipeline_id, void* state_arena, void* stash_arena,
                        void* work_arena, void* hip_stream, rc_stage** out) {
  const bool dry = !state_arena && !stash_arena && !work_arena;
  if (!dry) {
    if (!state_arena || !stash_arena || !work_arena)
      return fail(RC_ERR_INVALID_ARG, "either all three arenas or none (dry run)");
    if (((uintptr_t)state_arena | (uintptr_t)stash_arena | (uintptr_t)work_arena) % kAlign)
      return fail(RC_ERR_INVALID_ARG, "arenas must be 256-byte aligned");
  }
  rc_stage* st = new rc_stage();
  st->cfg = *cfg;
  st->adam = *adam;
  st->stage_index = stage_index;
  st->pipeline_id = pipeline_id;
  st->dry = dry;
  st->stream = (hipStream_t)hip_stream;
  st->state = (char*)state_arena;
  st->stash = (char*)stash_arena;
  st->work = (char*)work_arena;
  st->lay = y;
  for (int i = 0; i < RC_K_COUNT; ++i) st->stats[i] = {i, 0, 0.0, 0.0, 0.0};
  for (int i = 0; i < y.wslots; ++i) st->free_w.push_back(i);
  for (int i = 0; i < y.fslots; ++i) st->free_f.push_back(i);
  if (!dry) {
    hipError_t e = hipMemsetAsync(st->state, 0, y.state_bytes, st->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(st->stream);
    if (e != hipSuccess) {
      delete st;
      return fail(RC_ERR_HIP, std::string("zeroing the state arena: ") + hipGetErrorString(e));
    }
  }
  *out = st;
  return RC_OK;
}

}  // namespace

extern "C" {

rc_status rc_stage_memory_requirements(const rc_stage_config* cfg, size_t* state_bytes,
                                       size_t* stash_bytes, size_t* work_bytes) {
  if (!state_bytes || !stash_bytes || !work_bytes) return fail(RC_ERR_INVALID_ARG, "null output pointer");
  Layout y;
  rc_status r = make_layout(cfg, y);
  if (r != RC_OK) return r;
  *state_bytes = y.state_bytes;
  *stash_bytes = y.stash_bytes;
  *work_bytes = y.work_bytes;
  return RC_OK;
}

rc_status rc_stage_create(const rc_stage_config* cfg, const rc_adam_config* adam,
                          int32_t stage_index, int32_t pipeline_id, void* state_arena,
                          void* stash_arena, void* work_arena, void* hip_stream, rc_stage** out) {
  if (!out || !adam) return fail(RC_ERR_INVALID_ARG, "null argument");
  *out = nullptr;
  Layout y;
  rc_status r = make_layout(cfg, y);
  if (r != RC_OK) return r;
  return create_handle(y, cfg, adam, stage_index, pipeline_id, state_arena, stash_arena, work_arena,
                       hip_stream, out);
}

rc_status rc_stage_create_static(const rc_stage_config* cfg, const rc_adam_config* adam,
                                 int32_t stage_index, int32_t pipeline_id, void* state_arena,
                                 void* stash_arena, void* hip_stream, rc_stage** out) {
  if (!out || !adam) return fail(RC_ERR_INVALID_ARG, "null argument");
  *out = nullptr;
  Layout y;
  rc_status r = make_layout(cfg, y);
  if (r != RC_OK) return r;
  if (y.work_bytes > kScratchBytes)
    return fail(RC_ERR_UNSUPPORTED, "the configuration needs " + std::to_string(y.work_bytes) +
                                        " bytes of work memory; the no-allocation work memory holds " +
                                        std::to_string(kScratchBytes));
  if (!state_arena || !stash_arena) return fail(RC_ERR_INVALID_ARG, "null state or stash arena");
  void* work = nullptr;
  r = scratch_address((hipStream_t)hip_stream, &work);
  if (r != RC_OK) return r;
  return create_handle(y, cfg, adam, stage_index, pipeline_id, state_arena, stash_arena, work, hip_stream,
                       out);
}

rc_status rc_stage_destroy(rc_stage* st) {
  if (!st) return fail(RC_ERR_INVALID_ARG, "null stage");
  hipError_t e = st->dry ? hipSuccess : hipStreamSynchronize(st->stream);
  for (auto& r : st->pending) {
    st->pool.push_back(r.a);
    st->pool.push_back(r.b);
  }
  for (hipEvent_t ev : st->pool) hipEventDestroy(ev);
  delete st;
  if (e != hipSuccess) return fail(RC_ERR_HIP, std::string("destroy: ") + hipGetErrorString(e));
  return RC_OK;
}

rc_status rc_stage_load_param(rc_stage* st, int32_t layer, int32_t param_id, const float* host_src) {
  rc_status r = check_param(st, layer, param_id);
  if (r != RC_OK) return r;
  if (!host_src) return fail(RC_ERR_INVALID_ARG, "null host_src");
  const PLoc& p = st->lay.p[layer][param_id];
  float* dst = master(st, layer, param_id);
  HIPCHK(hipMemcpyAsync(dst, host_src, 4 * p.count, hipMemcpyHostToDevice, st->stream));
  const bool matrix = param_id == RC_P_W_QKV || param_id == RC_P_W_O || param_id == RC_P_W_1 ||
                      param_id == RC_P_W_2;
  if (st->lay.bf && matrix)
    HIPCHK(cast_f32_to_bf16(dst, (char*)st->state + st->lay.off_wb + 2 * p.off, p.count, st->stream));
  HIPCHK(hipStreamSynchronize(st->stream));
  st->can_rollback = false;  // the step's inverse no longer applies to replaced values
  return RC_OK;
}

rc_status rc_stage_read(rc_stage* st, int32_t what, int32_t layer, int32_t param_id, float* host_dst) {
  rc_status r = check_param(st, layer, param_id);
  if (r != RC_OK) return r;
  if (!host_dst) return fail(RC_ERR_INVALID_ARG, "null host_dst");
  size_t base;
  switch (what) {
    case RC_READ_PARAM: base = st->lay.off_master; break;
    case RC_READ_GRAD: base = st->lay.off_grad; break;
    case RC_READ_ADAM_M: base = st->lay.off_m; break;
    case RC_READ_ADAM_V: base = st->lay.off_v; break;
    default: return fail(RC_ERR_INVALID_ARG, "unknown read target");
  }
  const PLoc& p = st->lay.p[layer][param_id];
  HIPCHK(hipMemcpyAsync(host_dst, (float*)(st->state + base) + p.off, 4 * p.count,
                        hipMemcpyDeviceToHost, st->stream));
  HIPCHK(hipStreamSynchronize(st->stream));
  return RC_OK;
}

rc_status rc_stage_forward(rc_stage* st, rc_mb mb, const void* x, void* y) {
  if (!st) return fail(RC_ERR_INVALID_ARG, "null stage");
  if (!st->dry && (!x || !y || x == y)) return fail(RC_ERR_INVALID_ARG, "x, y must be distinct device buffers");
  auto key = std::make_pair(mb.j, mb.k);
  if (st->mbs.count(key))
    return fail(RC_ERR_BAD_STATE, "forward of micro-batch (" + std::to_string(mb.j) + "," +
                                      std::to_string(mb.k) + ") already ran this iteration");
  if (st->free_w.empty() || st->free_f.empty())
    return fail(RC_ERR_OUT_OF_STASH, "no free stash slot for micro-batch (" + std::to_string(mb.j) +
                                         "," + std::to_string(mb.k) + ")");
  if (st->limit && st->live + st->lay.acct_af > st->limit)
    return fail(RC_ERR_OUT_OF_STASH, "forward of micro-batch (" + std::to_string(mb.j) + "," +
                                         std::to_string(mb.k) + ") would exceed the stash limit");
  int ws = take_min(st->free_w), fs = take_min(st->free_f);
  if (!st->dry) {
    rc_status r = run_forward(st, ws, fs, x, y);
    if (r != RC_OK) {
      st->free_w.push_back(ws);
      st->free_f.push_back(fs);
      return r;
    }
  }
  st->mbs[key] = {1, ws, fs};
  st->live += st->lay.acct_af;
  st->peak = std::max(st->peak, st->live);
  record(st, RC_OP_F, mb.j, mb.k);
  st->closed = false;
  st->can_rollback = false;
  return RC_OK;
}

rc_status rc_stage_backward_input(rc_stage* st, rc_mb mb, const void* dy, void* dx) {
  if (!st) return fail(RC_ERR_INVALID_ARG, "null stage");
  if (!st->dry && (!dy || !dx || dy == dx)) return fail(RC_ERR_INVALID_ARG, "dy, dx must be distinct device buffers");
  auto it = st->mbs.find(std::make_pair(mb.j, mb.k));
  if (it == st->mbs.end() || it->second.state != 1)
    return fail(RC_ERR_BAD_STATE, "backward_input of micro-batch (" + std::to_string(mb.j) + "," +
                                      std::to_string(mb.k) + ") needs a completed forward and no prior B");
  if (!st->dry) {
    rc_status r = run_backward_input(st, it->second.ws, it->second.fs, dy, dx);
    if (r != RC_OK) return r;
  }
  st->free_f.push_back(it->second.fs);
  it->second.fs = -1;
  it->second.state = 2;
  st->live += st->lay.acct_sw - st->lay.acct_af;
  st->peak = std::max(st->peak, st->live);
  record(st, RC_OP_B, mb.j, mb.k);
  st->closed = false;
  st->can_rollback = false;
  return RC_OK;
}

rc_status rc_stage_backward(rc_stage* st, rc_mb mb, const void* dy, void* dx) {
  if (!st) return fail(RC_ERR_INVALID_ARG, "null stage");
  if (!st->dry && (!dy || !dx || dy == dx)) return fail(RC_ERR_INVALID_ARG, "dy, dx must be distinct device buffers");
  auto it = st->mbs.find(std::make_pair(mb.j, mb.k));
  if (it == st->mbs.end() || it->second.state != 1)
    return fail(RC_ERR_BAD_STATE, "backward of micro-batch (" + std::to_string(mb.j) + "," +
                                      std::to_string(mb.k) + ") needs a completed forward and no prior B");
  if (!st->dry) {
    rc_status r = run_backward_input(st, it->second.ws, it->second.fs, dy, dx);
    if (r != RC_OK) return r;
    const int ws = it->second.ws;
    r = run_backward_weight(st, &ws, 1);
    if (r != RC_OK) return r;
  }
  st->free_f.push_back(it->second.fs);
  st->free_w.push_back(it->second.ws);
  it->second.fs = -1;
  it->second.ws = -1;
  it->second.state = 3;
  st->live -= st->lay.acct_af;
  record(st, RC_OP_B, mb.j, mb.k);
  record(st, RC_OP_W, mb.j, mb.k);
  st->grads_fresh = false;
  st->closed = false;
  st->can_rollback = false;
  return RC_OK;
}

rc_status rc_stage_stash_account(rc_stage* st, rc_stash_account* out, int32_t reset_peak) {
  if (!st || !out) return fail(RC_ERR_INVALID_ARG, "bad stash_account arguments");
  if (reset_peak) st->peak = st->live;
  out->a_f = st->lay.acct_af;
  out->s_w = st->lay.acct_sw;
  out->live = st->live;
  out->peak = st->peak;
  out->limit = st->limit;
  return RC_OK;
}

rc_status rc_stage_set_stash_limit(rc_stage* st, uint64_t bytes) {
  if (!st) return fail(RC_ERR_INVALID_ARG, "null stage");
  if (bytes && bytes < st->lay.acct_af)
    return fail(RC_ERR_INVALID_ARG, "a stash limit below one micro-batch's forward share admits no forward");
  st->limit = bytes;
  return RC_OK;
}

rc_status rc_stage_backward_weight_many(rc_stage* st, const rc_mb* mbs, int32_t n) {
  if (!st) return fail(RC_ERR_INVALID_ARG, "null stage");
  if (n < 1 || n > GEMM_MAX_SEG || !mbs)
    return fail(RC_ERR_INVALID_ARG, "need 1 <= n <= " + std::to_string(GEMM_MAX_SEG) + " micro-batches");
  int ws[GEMM_MAX_SEG];
  std::vector<std::pair<int, int>> keys;
  for (int q = 0; q < n; ++q) {
    auto key = std::make_pair(mbs[q].j, mbs[q].k);
    auto it = st->mbs.find(key);
    if (it == st->mbs.end() || it->second.state != 2)
      return fail(RC_ERR_BAD_STATE, "backward_weight of micro-batch (" + std::to_string(mbs[q].j) + "," +
                                        std::to_string(mbs[q].k) + ") needs a completed B and no prior W");
    if (std::find(keys.begin(), keys.end(), key) != keys.end())
      return fail(RC_ERR_BAD_STATE, "micro-batch (" + std::to_string(mbs[q].j) + "," +
                                        std::to_string(mbs[q].k) + ") listed twice");
    keys.push_back(key);
    ws[q] = it->second.ws;
  }
  if (!st->dry) {
    rc_status r = run_backward_weight(st, ws, n);
    if (r != RC_OK) return r;
  }
  for (int q = 0; q < n; ++q) {
    MbRec& m = st->mbs[keys[q]];
    st->live -= st->lay.acct_sw;
    st->free_w.push_back(m.ws);
    m.ws = -1;
    m.state = 3;
    record(st, RC_OP_W, mbs[q].j, mbs[q].k);
    st->closed = false;
    st->can_rollback = false;
  }
  st->grads_fresh = false;
  return RC_OK;
}

rc_status rc_stage_backward_weight(rc_stage* st, rc_mb mb) { return rc_stage_backward_weight_many(st, &mb, 1); }

rc_status rc_stage_optimizer_step(rc_stage* st, float grad_scale) {
  if (!st) return fail(RC_ERR_INVALID_ARG, "null stage");
  for (auto& kv : st->mbs)
    if (kv.second.state != 3)
      return fail(RC_ERR_BAD_STATE, "optimizer step while micro-batch (" +
                                        std::to_string(kv.first.first) + "," +
                                        std::to_string(kv.first.second) + ") has not run W");
  if (!st->dry) {
    rc_status r = run_optimizer(st, grad_scale);
    if (r != RC_OK) return r;
  }
  st->t += 1;
  record(st, RC_OP_STEP, -1, -1);
  st->mbs.clear();
  st->grads_fresh = true;
  st->iter += 1;
  st->closed = true;
  st->can_rollback = true;
  st->last_scale = grad_scale;
  return RC_OK;
}

rc_status rc_stage_optimizer_skip(rc_stage* st) {
  if (!st) return fail(RC_ERR_INVALID_ARG, "null stage");
  for (auto& kv : st->mbs)
    if (kv.second.state != 3)
      return fail(RC_ERR_BAD_STATE, "optimizer skip while micro-batch (" +
                                        std::to_string(kv.first.first) + "," +
                                        std::to_string(kv.first.second) + ") has not run W");
  // the gradient of an iteration without a weight pass is zero (as a step would use it)
  if (!st->dry && st->grads_fresh)
    HIPCHK(fill_f32((float*)(st->state + st->lay.off_grad), st->lay.n_total, 0.f, st->stream));
  record(st, RC_OP_SKIP, -1, -1);
  st->mbs.clear();
  st->grads_fresh = true;
  st->iter += 1;
  st->closed = true;
  st->can_rollback = false;
  return RC_OK;
}

rc_status rc_stage_optimizer_rollback(rc_stage* st) {
  if (!st) return fail(RC_ERR_INVALID_ARG, "null stage");
  if (!st->can_rollback) return fail(RC_ERR_BAD_STATE, "rollback needs an optimizer step as the last call");
  if (!st->dry) {
    rc_status r = run_rollback(st);
    if (r != RC_OK) return r;
  }
  st->t -= 1;
  record(st, RC_OP_ROLLBACK, -1, -1);
  st->log.back().iter = st->iter - 1;  // the iteration whose step is undone
  st->can_rollback = false;
  return RC_OK;
}

rc_status rc_stage_grad_check(rc_stage* st, float grad_scale, double* sumsq, int64_t* nonfinite) {
  if (!st || !sumsq || !nonfinite) return fail(RC_ERR_INVALID_ARG, "bad grad_check arguments");
  *sumsq = 0.0;
  *nonfinite = 0;
  if (st->grads_fresh && !st->closed) return RC_OK;  // no weight pass yet: zero gradient
  if (st->dry) return fail(RC_ERR_INVALID_ARG, "dry-run handle has no device memory");
  const Layout& y = st->lay;
  float* part = (float*)(st->work + y.off_check);
  int* bad = (int*)(part + GRAD_CHECK_BLOCKS);
  HIPCHK(grad_check((const float*)(st->state + y.off_grad), y.n_total, grad_scale, part, bad, st->stream));
  std::vector<float> hp(GRAD_CHECK_BLOCKS);
  std::vector<int> hb(GRAD_CHECK_BLOCKS);
  HIPCHK(hipMemcpyAsync(hp.data(), part, 4 * GRAD_CHECK_BLOCKS, hipMemcpyDeviceToHost, st->stream));
  HIPCHK(hipMemcpyAsync(hb.data(), bad, 4 * GRAD_CHECK_BLOCKS, hipMemcpyDeviceToHost, st->stream));
  HIPCHK(hipStreamSynchronize(st->stream));
  double s = 0.0;
  int64_t b = 0;
  for (int i = 0; i < GRAD_CHECK_BLOCKS; ++i) {
    s += hp[i];
    b += hb[i];
  }
  *sumsq = s;
  *nonfinite = b;
  return RC_OK;
}

rc_status rc_stage_op_log(rc_stage* st, rc_op_record* buf, int32_t cap, int32_t* n) {
  if (!st || !n || (cap > 0 && !buf) || cap < 0) return fail(RC_ERR_INVALID_ARG, "bad op_log arguments");
  *n = (int32_t)st->log.size();
  const int32_t m = std::min<int32_t>(cap, *n);
  if (m > 0) std::memcpy(buf, st->log.data(), sizeof(rc_op_record) * m);
  return RC_OK;
}

rc_status rc_stage_stash_usage(rc_stage* st, int32_t* stashed, int32_t* inflight) {
  if (!st || !stashed || !inflight) return fail(RC_ERR_INVALID_ARG, "null argument");
  *stashed = st->lay.wslots - (int32_t)st->free_w.size();
  *inflight = st->lay.fslots - (int32_t)st->free_f.size();
  return RC_OK;
}

rc_status rc_stage_set_stream(rc_stage* st, void* hip_stream) {
  if (!st) return fail(RC_ERR_INVALID_ARG, "null stage");
  st->stream = (hipStream_t)hip_stream;
  return RC_OK;
}

rc_status rc_stage_attention_kernels(rc_stage* st, int32_t* kind) {
  if (!st || !kind) return fail(RC_ERR_INVALID_ARG, "null argument");
  const Layout& y = st->lay;
  if (!y.flash) *kind = RC_ATTN_MATERIALISED;
  else *kind = y.causal && attn_flash_paired(y.b, y.s, y.a) ? RC_ATTN_PAIRED : RC_ATTN_BLOCK;
  return RC_OK;
}

rc_status rc_stage_synchronize(rc_stage* st) {
  if (!st) return fail(RC_ERR_INVALID_ARG, "null stage");
  if (st->dry) return RC_OK;
  HIPCHK(hipStreamSynchronize(st->stream));
  HIPCHK(hipGetLastError());
  return RC_OK;
}

rc_status rc_stage_profile_enable(rc_stage* st, int32_t enable) {
  if (!st || st->dry) return fail(RC_ERR_INVALID_ARG, "profiling needs a device handle");
  if (enable) {
    HIPCHK(hipStreamSynchronize(st->stream));
    for (auto& r : st->pending) {
      st->pool.push_back(r.a);
      st->pool.push_back(r.b);
    }
    st->pending.clear();
    for (int i = 0; i < RC_K_COUNT; ++i) st->stats[i] = {i, 0, 0.0, 0.0, 0.0};
  }
  st->prof = enable != 0;
  return RC_OK;
}

rc_status rc_stage_profile_read(rc_stage* st, rc_kernel_stat* out) {
  if (!st || st->dry || !out) return fail(RC_ERR_INVALID_ARG, "profiling needs a device handle");
  HIPCHK(hipStreamSynchronize(st->stream));
  for (auto& r : st->pending) {
    float ms = 0.f;
    HIPCHK(hipEventElapsedTime(&ms, r.a, r.b));
    rc_kernel_stat& k = st->stats[r.kind];
    k.launches += 1;
    k.ms += ms;
    k.flops += r.flops;
    k.bytes += r.bytes;
    st->pool.push_back(r.a);
    st->pool.push_back(r.b);
  }
  st->pending.clear();
  for (int i = 0; i < RC_K_COUNT; ++i) out[i] = st->stats[i];
  return RC_OK;
}

const char* rc_last_error(void) { return g_err.c_str(); }

}  // extern "C"

// Shared with the planner's translation unit: set the thread-local message.
rc_status rc_set_error(rc_status s, const std::string& msg) { return fail(s, msg); }
