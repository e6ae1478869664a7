"""fp64 CPU oracle of one ReCycle pipeline stage (plain numpy).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only the tests, the package's smoke check and the
benchmark's CPU-baseline leg use it.  It shares no code with the HIP path; the
two meet only through the seeded inputs of ``synth``.

What it computes (Gandhi et al., "ReCycle", SOSP'24):

* One pipeline stage = L pre-LN GPT transformer layers (the evaluation trains
  Megatron GPT-3 with TP = 1, Evaluation section, Workloads paragraph).
* Decoupled BackProp (section 3.2 and the forward/backward-of-an-operator
  figure): the backward pass has two outputs, the gradient w.r.t. the stage
  input (B_input) and the gradients w.r.t. the parameters (B_weight).  B_input
  is all the upstream stage needs; B_weight has no consumer inside the
  iteration and can run later, in any order, from stored intermediates (the
  WeightGradStore of section 5).
* Gradient accumulation over the stage's own and re-routed micro-batches
  (Adaptive Pipelining, section 3.1): peers hold identical parameters, so a
  re-routed micro-batch contributes exactly what it would have on its own
  pipeline; the math of the iteration is unchanged.
* Staggered Optimizer (section 3.3): each stage's AdamW step (section 5,
  post-step validation paragraph) depends only on that stage's own gradients.
* Op identity (i, j, k, c, k_s) of the MILP notation (section 4.2.2): stage,
  micro-batch, original pipeline, op type, executing pipeline; and the
  same-stage dependency B_input -> B_weight (same-stage constraint equation).

Readings of points the paper leaves open (pre-LN GPT block, biases on all four
linears, LN with affine, tanh GeLU, LN eps 1e-5 with biased variance, scale
1/sqrt(d), causal mask with -inf, no dropout, W stored [in, out], fused QKV with
column blocks Q|K|V, AdamW hyper-parameters) are listed in the design notes
and mirrored here.

Every function below is pinned by ``tests/test_oracle_pins.py`` (finite
differences, an independent torch fp64 autograd build of the same block,
closed forms and invariants).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Optional, Tuple

import numpy as np

F64 = np.float64

# ---------------------------------------------------------------------------
# Elementary operations
# ---------------------------------------------------------------------------


def layer_norm(z: np.ndarray, g: np.ndarray, b: np.ndarray, eps: float):
    """LN(z) = (z - mean) * (var + eps)^(-1/2) * g + b over the last axis.

    Biased variance (divide by h).  Returns (out, zhat, rstd)."""
    mu = z.mean(axis=-1, keepdims=True)
    var = ((z - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    zhat = (z - mu) * rstd
    return zhat * g + b, zhat, rstd


def layer_norm_grad_input(dout: np.ndarray, zhat: np.ndarray, rstd: np.ndarray, g: np.ndarray):
    """Vector-Jacobian product of LN w.r.t. its input z."""
    dzhat = dout * g
    h = zhat.shape[-1]
    return rstd * (dzhat - dzhat.sum(-1, keepdims=True) / h
                   - zhat * (dzhat * zhat).sum(-1, keepdims=True) / h)


_GELU_C = np.sqrt(2.0 / np.pi)


def gelu(u: np.ndarray) -> np.ndarray:
    """tanh form of GeLU: 0.5 u (1 + tanh(sqrt(2/pi) (u + 0.044715 u^3)))."""
    return 0.5 * u * (1.0 + np.tanh(_GELU_C * (u + 0.044715 * u ** 3)))


def gelu_prime(u: np.ndarray) -> np.ndarray:
    t = np.tanh(_GELU_C * (u + 0.044715 * u ** 3))
    return 0.5 * (1.0 + t) + 0.5 * u * (1.0 - t * t) * _GELU_C * (1.0 + 3 * 0.044715 * u * u)


def softmax_rows(s: np.ndarray) -> np.ndarray:
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=-1, keepdims=True)


def attention(q, k, v, causal: bool):
    """Scaled dot-product attention per (sequence, head).

    q, k, v: [b, a, s, d].  Scores S = q k^T / sqrt(d); with ``causal`` the
    entries S[i, j > i] are -inf so their probabilities are exactly 0.
    Returns (o [b, a, s, d], p [b, a, s, s])."""
    d = q.shape[-1]
    s = np.matmul(q, np.swapaxes(k, -1, -2)) / np.sqrt(d)
    if causal:
        n = s.shape[-1]
        s = np.where(np.triu(np.ones((n, n), dtype=bool), 1), -np.inf, s)
    p = softmax_rows(s)
    return np.matmul(p, v), p


def attention_grad(do, q, k, v, p):
    """VJP of ``attention`` given the saved probabilities p."""
    d = q.shape[-1]
    dv = np.matmul(np.swapaxes(p, -1, -2), do)
    dp = np.matmul(do, np.swapaxes(v, -1, -2))
    ds = p * (dp - (dp * p).sum(-1, keepdims=True)) / np.sqrt(d)
    dq = np.matmul(ds, k)
    dk = np.matmul(np.swapaxes(ds, -1, -2), q)
    return dq, dk, dv


def split_heads(qkv: np.ndarray, heads: int):
    """[b, s, 3h] -> three [b, a, s, d]; head n of Q uses columns n*d..(n+1)*d-1."""
    b, s, h3 = qkv.shape
    h = h3 // 3
    d = h // heads
    x = qkv.reshape(b, s, 3, heads, d)
    return (np.ascontiguousarray(x[:, :, 0].transpose(0, 2, 1, 3)),
            np.ascontiguousarray(x[:, :, 1].transpose(0, 2, 1, 3)),
            np.ascontiguousarray(x[:, :, 2].transpose(0, 2, 1, 3)))


def to_heads(x: np.ndarray, heads: int) -> np.ndarray:
    """[b, s, a*d] -> [b, a, s, d]."""
    b, s, h = x.shape
    return np.ascontiguousarray(x.reshape(b, s, heads, h // heads).transpose(0, 2, 1, 3))


def merge_heads(x: np.ndarray) -> np.ndarray:
    """[b, a, s, d] -> [b, s, a*d]."""
    b, a, s, d = x.shape
    return np.ascontiguousarray(x.transpose(0, 2, 1, 3)).reshape(b, s, a * d)


def _tok(x: np.ndarray) -> np.ndarray:
    """[b, s, n] -> [b*s, n] (token-major matrix)."""
    return x.reshape(-1, x.shape[-1])


# ---------------------------------------------------------------------------
# One pre-LN transformer layer
# ---------------------------------------------------------------------------


@dataclass
class LayerShape:
    heads: int
    causal: bool
    eps: float


def layer_forward(x, P, shp: LayerShape):
    """Forward of one pre-LN GPT layer.  P = 12 params in synth.PARAM_NAMES order.

    A = LN1(X); [Q|K|V] = A W_qkv + b_qkv; O = attn(Q, K, V);
    H = X + O W_o + b_o; C = LN2(H); U = C W_1 + b_1; G = gelu(U);
    Y = H + G W_2 + b_2.  Returns (Y, cache)."""
    g1, be1, wqkv, bqkv, wo, bo, g2, be2, w1, b1, w2, b2 = P
    A, xhat1, r1 = layer_norm(x, g1, be1, shp.eps)
    qkv = A @ wqkv + bqkv
    q, k, v = split_heads(qkv, shp.heads)
    oh, p = attention(q, k, v, shp.causal)
    O = merge_heads(oh)
    H = x + O @ wo + bo
    C, xhat2, r2 = layer_norm(H, g2, be2, shp.eps)
    U = C @ w1 + b1
    G = gelu(U)
    Y = H + G @ w2 + b2
    cache = dict(A=A, xhat1=xhat1, r1=r1, q=q, k=k, v=v, p=p, O=O,
                 C=C, xhat2=xhat2, r2=r2, U=U, G=G)
    return Y, cache


def layer_backward_fused(dY, cache, P):
    """Conventional (coupled) reverse pass: returns (dX, grads) together."""
    g1, be1, wqkv, bqkv, wo, bo, g2, be2, w1, b1, w2, b2 = P
    c = cache
    grads = [None] * 12
    # FC2 + residual
    grads[10] = _tok(c["G"]).T @ _tok(dY)
    grads[11] = _tok(dY).sum(0)
    dU = (dY @ w2.T) * gelu_prime(c["U"])
    grads[8] = _tok(c["C"]).T @ _tok(dU)
    grads[9] = _tok(dU).sum(0)
    dC = dU @ w1.T
    grads[6] = _tok(dC * c["xhat2"]).sum(0)
    grads[7] = _tok(dC).sum(0)
    dH = dY + layer_norm_grad_input(dC, c["xhat2"], c["r2"], g2)
    grads[4] = _tok(c["O"]).T @ _tok(dH)
    grads[5] = _tok(dH).sum(0)
    dO = to_heads(dH @ wo.T, c["q"].shape[1])
    dq, dk, dv = attention_grad(dO, c["q"], c["k"], c["v"], c["p"])
    dQKV = np.concatenate([merge_heads(dq), merge_heads(dk), merge_heads(dv)], axis=-1)
    grads[2] = _tok(c["A"]).T @ _tok(dQKV)
    grads[3] = _tok(dQKV).sum(0)
    dA = dQKV @ wqkv.T
    grads[0] = _tok(dA * c["xhat1"]).sum(0)
    grads[1] = _tok(dA).sum(0)
    dX = dH + layer_norm_grad_input(dA, c["xhat1"], c["r1"], g1)
    return dX, grads


def layer_backward_input(dY, cache, P):
    """B_input of one layer: the input gradient dX only.

    No parameter gradient is formed.  Returns (dX, wstash) where wstash holds
    exactly the operand pairs the deferred weight pass needs: (A, dQKV),
    (O, dH), (C, dU), (G, dY) for the four linears and (xhat, dLNout) for the
    two LayerNorms."""
    g1, be1, wqkv, bqkv, wo, bo, g2, be2, w1, b1, w2, b2 = P
    c = cache
    dU = (dY @ w2.T) * gelu_prime(c["U"])
    dC = dU @ w1.T
    dH = dY + layer_norm_grad_input(dC, c["xhat2"], c["r2"], g2)
    dO = to_heads(dH @ wo.T, c["q"].shape[1])
    dq, dk, dv = attention_grad(dO, c["q"], c["k"], c["v"], c["p"])
    dQKV = np.concatenate([merge_heads(dq), merge_heads(dk), merge_heads(dv)], axis=-1)
    dA = dQKV @ wqkv.T
    dX = dH + layer_norm_grad_input(dA, c["xhat1"], c["r1"], g1)
    wstash = dict(A=c["A"], dQKV=dQKV, O=c["O"], dH=dH, C=c["C"], dU=dU,
                  G=c["G"], dY=dY, xhat1=c["xhat1"], dA=dA, xhat2=c["xhat2"], dC=dC)
    return dX, wstash


def layer_backward_weight(ws) -> List[np.ndarray]:
    """B_weight of one layer from its stash: dW = X^T dY per linear, column
    sums for biases, sum(dLNout * xhat) and sum(dLNout) for LN affine."""
    t = _tok
    return [
        t(ws["dA"] * ws["xhat1"]).sum(0), t(ws["dA"]).sum(0),
        t(ws["A"]).T @ t(ws["dQKV"]), t(ws["dQKV"]).sum(0),
        t(ws["O"]).T @ t(ws["dH"]), t(ws["dH"]).sum(0),
        t(ws["dC"] * ws["xhat2"]).sum(0), t(ws["dC"]).sum(0),
        t(ws["C"]).T @ t(ws["dU"]), t(ws["dU"]).sum(0),
        t(ws["G"]).T @ t(ws["dY"]), t(ws["dY"]).sum(0),
    ]


# ---------------------------------------------------------------------------
# Whole stage
# ---------------------------------------------------------------------------


def stage_forward(x, params, shp: LayerShape):
    caches = []
    for P in params:
        x, c = layer_forward(x, P, shp)
        caches.append(c)
    return x, caches


def stage_backward_fused(dy, caches, params):
    grads = [None] * len(params)
    for l in reversed(range(len(params))):
        dy, grads[l] = layer_backward_fused(dy, caches[l], params[l])
    return dy, grads


def stage_backward_input(dy, caches, params):
    stashes = [None] * len(params)
    for l in reversed(range(len(params))):
        dy, stashes[l] = layer_backward_input(dy, caches[l], params[l])
    return dy, stashes


def stage_backward_weight(stashes):
    return [layer_backward_weight(ws) for ws in stashes]


# ---------------------------------------------------------------------------
# AdamW (Kingma & Ba bias correction, Loshchilov & Hutter decoupled decay)
# ---------------------------------------------------------------------------


@dataclass
class AdamHP:
    lr: float = 1e-4
    beta1: float = 0.9
    beta2: float = 0.95
    eps: float = 1e-8
    weight_decay: float = 0.1


def adamw_update(p, g, m, v, t: int, hp: AdamHP, decay: bool):
    """One AdamW step at step number t (1-based); returns new (p, m, v).

    m <- b1 m + (1-b1) g;  v <- b2 v + (1-b2) g^2;
    p <- p (1 - lr wd) - lr * (m / (1-b1^t)) / (sqrt(v / (1-b2^t)) + eps)."""
    m = hp.beta1 * m + (1.0 - hp.beta1) * g
    v = hp.beta2 * v + (1.0 - hp.beta2) * g * g
    mhat = m / (1.0 - hp.beta1 ** t)
    vhat = v / (1.0 - hp.beta2 ** t)
    wd = hp.weight_decay if decay else 0.0
    p = p * (1.0 - hp.lr * wd) - hp.lr * mhat / (np.sqrt(vhat) + hp.eps)
    return p, m, v


def adamw_rollback(p, g, m, v, t: int, hp: AdamHP, decay: bool):
    """Undo the AdamW step number t: from the stepped (p, m, v) and the gradient g
    that step used, the values before it.  No copy of the old state is needed
    because every assignment of the step is invertible (section 5, post-step
    validation paragraph: a rollback costs no extra memory for AdamW).

    The assignments of ``adamw_update`` are undone in reverse order: the
    parameter update used the new m and v, so p is restored first, then
    v <- (v - (1-b2) g^2) / b2 and m <- (m - (1-b1) g) / b1."""
    mhat = m / (1.0 - hp.beta1 ** t)
    vhat = v / (1.0 - hp.beta2 ** t)
    wd = hp.weight_decay if decay else 0.0
    p = (p + hp.lr * mhat / (np.sqrt(vhat) + hp.eps)) / (1.0 - hp.lr * wd)
    if t == 1:  # the moments before the first step are the zero initial state
        return p, np.zeros_like(m), np.zeros_like(v)
    v = (v - (1.0 - hp.beta2) * g * g) / hp.beta2
    m = (m - (1.0 - hp.beta1) * g) / hp.beta1
    return p, m, v


# ---------------------------------------------------------------------------
# Stage object with the micro-batch state machine and op log
# ---------------------------------------------------------------------------

OP_F, OP_B, OP_W, OP_STEP, OP_SKIP, OP_ROLLBACK = 0, 1, 2, 3, 4, 5
MATRIX_IDS = (2, 4, 8, 10)


def stash_bytes(cfg, fused_attention: bool):
    """Bytes one micro-batch holds between its calls (all layers): (a_f, s_w).

    The memory change of each op in the schedule MILP (section 4.2.2), read
    as F: +a_f, B_input: +(s_w - a_f), B_weight: -s_w (the printed cases do
    not net to zero per micro-batch; this reading does).  a_f is what the
    backward passes need from the forward pass: per layer A, LN1 input X, Q, K,
    V, O, H, C, U, G (8 T h + 2 T f elements), the LayerNorm mean and rstd
    (4 fp32 per token) and the attention's kept state: the probabilities
    (b heads s^2 elements) or, with fused attention, the row log-sum-exp
    (b heads s fp32).  s_w is what the deferred weight pass needs: the
    operand pairs of the four linears and the two LayerNorms, 12 T h + 2 T f
    elements, plus the LayerNorm statistics.  E = 2 (bf16) or 4 (fp32)."""
    E = 2 if cfg.dtype == "bf16" else 4
    T = cfg.micro_batch * cfg.seq
    h, f = cfg.hidden, cfg.ffn
    rows = cfg.micro_batch * cfg.heads * cfg.seq
    attn = 4 * rows if fused_attention else E * rows * cfg.seq
    a_f = cfg.layers * (E * (8 * T * h + 2 * T * f) + 16 * T + attn)
    s_w = cfg.layers * (E * (12 * T * h + 2 * T * f) + 16 * T)
    return a_f, s_w


class StageError(Exception):
    """code is one of 'BAD_STATE', 'OUT_OF_STASH', 'INVALID_ARG'."""

    def __init__(self, code: str, msg: str):
        super().__init__(f"{code}: {msg}")
        self.code = code


class OracleStage:
    """One pipeline stage i on data-parallel pipeline k_s.

    Per micro-batch (j, k) and iteration: EMPTY -F-> F_DONE -B-> B_DONE -W->
    DONE.  B before F, W before B, F or B twice are BAD_STATE; the optimizer
    step is BAD_STATE while any micro-batch of the iteration is not DONE.
    Post-step validation (section 5): ``grad_check`` reports the squared norm
    and the non-finite entries of the gradient; ``optimizer_skip`` closes the
    iteration without an update (a failed check here or upstream);
    ``optimizer_rollback`` undoes the step just taken (a failed check
    downstream), allowed only while no other call followed that step.
    ``max_stashed`` bounds micro-batches holding weight-pass intermediates
    (F..W), ``max_inflight`` those holding forward-only intermediates (F..B);
    exceeding either is OUT_OF_STASH.  Gradients are zeroed at the first W of
    an iteration, so the previous iteration's gradients stay readable until
    then."""

    def __init__(self, cfg, params, hp: Optional[AdamHP] = None, stage_index: int = 0,
                 pipeline_id: int = 0, max_stashed: Optional[int] = None,
                 max_inflight: Optional[int] = None):
        self.cfg = cfg
        self.shp = LayerShape(cfg.heads, cfg.causal, cfg.ln_eps)
        self.params = [[np.array(p, dtype=F64) for p in layer] for layer in params]
        self.grads = [[np.zeros_like(p) for p in layer] for layer in self.params]
        self.m = [[np.zeros_like(p) for p in layer] for layer in self.params]
        self.v = [[np.zeros_like(p) for p in layer] for layer in self.params]
        self.hp = hp or AdamHP()
        self.stage_index = stage_index
        self.pipeline_id = pipeline_id
        self.max_stashed = max_stashed if max_stashed is not None else cfg.stash_slots
        self.max_inflight = max_inflight if max_inflight is not None else cfg.inflight_slots
        self.t = 0
        self.iter = 0
        self.state: Dict[Tuple[int, int], str] = {}
        self.caches: Dict[Tuple[int, int], list] = {}
        self.wstash: Dict[Tuple[int, int], list] = {}
        self.grads_fresh = True
        self.log: List[Tuple[int, int, int, int, int, int]] = []
        self.closed = False          # the last call closed an iteration (step / skip / rollback)
        self.last_step_scale = None  # grad_scale of a step that may still be rolled back
        # stash accounting; the library keeps fused attention's row statistics
        # instead of probabilities for bf16 stages with head dimension 128
        fused = cfg.dtype == "bf16" and cfg.hidden // cfg.heads == 128
        self.a_f, self.s_w = stash_bytes(cfg, fused)
        self.live = self.peak = self.limit = 0

    # -- bookkeeping -------------------------------------------------------
    def _record(self, op, mb):
        j, k = (mb if mb is not None else (-1, -1))
        self.log.append((len(self.log), op, j, k, self.pipeline_id, self.iter))

    def _n_stashed(self):
        return sum(1 for s in self.state.values() if s in ("F", "B"))

    def _n_inflight(self):
        return sum(1 for s in self.state.values() if s == "F")

    # -- the four calls ------------------------------------------------------
    def forward(self, mb, x):
        mb = (int(mb[0]), int(mb[1]))
        if mb in self.state:
            raise StageError("BAD_STATE", f"forward of {mb} twice in iteration {self.iter}")
        if self._n_stashed() >= self.max_stashed or self._n_inflight() >= self.max_inflight:
            raise StageError("OUT_OF_STASH", f"no stash slot for {mb}")
        if self.limit and self.live + self.a_f > self.limit:
            raise StageError("OUT_OF_STASH", f"forward of {mb} would exceed the stash limit")
        y, caches = stage_forward(np.asarray(x, dtype=F64), self.params, self.shp)
        self.caches[mb] = caches
        self.state[mb] = "F"
        self.live += self.a_f
        self.peak = max(self.peak, self.live)
        self._record(OP_F, mb)
        self.closed = False
        self.last_step_scale = None
        return y

    def backward_input(self, mb, dy):
        mb = (int(mb[0]), int(mb[1]))
        if self.state.get(mb) != "F":
            raise StageError("BAD_STATE", f"backward_input of {mb} in state {self.state.get(mb)}")
        dx, stashes = stage_backward_input(np.asarray(dy, dtype=F64), self.caches.pop(mb), self.params)
        self.wstash[mb] = stashes
        self.state[mb] = "B"
        self.live += self.s_w - self.a_f
        self.peak = max(self.peak, self.live)
        self._record(OP_B, mb)
        self.closed = False
        self.last_step_scale = None
        return dx

    def backward_weight(self, mb):
        mb = (int(mb[0]), int(mb[1]))
        if self.state.get(mb) != "B":
            raise StageError("BAD_STATE", f"backward_weight of {mb} in state {self.state.get(mb)}")
        gs = stage_backward_weight(self.wstash.pop(mb))
        if self.grads_fresh:
            for layer in self.grads:
                for g in layer:
                    g[...] = 0.0
            self.grads_fresh = False
        for l, layer in enumerate(gs):
            for p, g in enumerate(layer):
                self.grads[l][p] += g
        self.state[mb] = "W"
        self.live -= self.s_w
        self._record(OP_W, mb)
        self.closed = False
        self.last_step_scale = None

    def backward(self, mb, dy):
        """Coupled backward: B_input then B_weight of mb (the peak counts the
        stash between calls, so the pair changes it by -a_f at once)."""
        mb = (int(mb[0]), int(mb[1]))
        if self.state.get(mb) != "F":
            raise StageError("BAD_STATE", f"backward of {mb} in state {self.state.get(mb)}")
        peak = self.peak
        dx = self.backward_input(mb, dy)
        self.backward_weight(mb)
        self.peak = peak
        return dx

    def stash_account(self, reset_peak: bool = False):
        if reset_peak:
            self.peak = self.live
        return {"a_f": self.a_f, "s_w": self.s_w, "live": self.live, "peak": self.peak,
                "limit": self.limit}

    def set_stash_limit(self, nbytes: int):
        if nbytes and nbytes < self.a_f:
            raise StageError("INVALID_ARG", "a stash limit below a_f admits no forward")
        self.limit = int(nbytes)

    def optimizer_step(self, grad_scale: float = 1.0):
        pending = [mb for mb, s in self.state.items() if s != "W"]
        if pending:
            raise StageError("BAD_STATE", f"optimizer step with pending micro-batches {pending}")
        if self.grads_fresh:  # no weight pass ran this iteration: zero gradient
            for layer in self.grads:
                for g in layer:
                    g[...] = 0.0
        self.t += 1
        for l in range(len(self.params)):
            for p in range(len(self.params[l])):
                self.params[l][p], self.m[l][p], self.v[l][p] = adamw_update(
                    self.params[l][p], grad_scale * self.grads[l][p], self.m[l][p],
                    self.v[l][p], self.t, self.hp, decay=p in MATRIX_IDS)
        self._record(OP_STEP, None)
        self.state.clear()
        self.grads_fresh = True
        self.iter += 1
        self.closed = True
        self.last_step_scale = grad_scale

    def optimizer_skip(self):
        """Close the iteration without an update."""
        pending = [mb for mb, s in self.state.items() if s != "W"]
        if pending:
            raise StageError("BAD_STATE", f"optimizer skip with pending micro-batches {pending}")
        if self.grads_fresh:
            for layer in self.grads:
                for g in layer:
                    g[...] = 0.0
        self._record(OP_SKIP, None)
        self.state.clear()
        self.grads_fresh = True
        self.iter += 1
        self.closed = True
        self.last_step_scale = None

    def optimizer_rollback(self):
        """Undo the step just taken, from the retained gradients."""
        if self.last_step_scale is None:
            raise StageError("BAD_STATE", "rollback needs an optimizer step as the last call")
        gs = self.last_step_scale
        for l in range(len(self.params)):
            for p in range(len(self.params[l])):
                self.params[l][p], self.m[l][p], self.v[l][p] = adamw_rollback(
                    self.params[l][p], gs * self.grads[l][p], self.m[l][p], self.v[l][p], self.t,
                    self.hp, decay=p in MATRIX_IDS)
        self.t -= 1
        self.log.append((len(self.log), OP_ROLLBACK, -1, -1, self.pipeline_id, self.iter - 1))
        self.last_step_scale = None

    def grad_check(self, grad_scale: float = 1.0):
        """(sum of squares, number of non-finite entries) of grad_scale * the
        gradient: the one being accumulated, or, right after the iteration
        closed, the one its step used (zero if no weight pass ran)."""
        if self.grads_fresh and not self.closed:
            return 0.0, 0
        ss, bad = 0.0, 0
        for layer in self.grads:
            for g in layer:
                x = grad_scale * g
                fin = np.isfinite(x)
                bad += int(x.size - fin.sum())
                ss += float(np.sum(x[fin] ** 2))
        return ss, bad
