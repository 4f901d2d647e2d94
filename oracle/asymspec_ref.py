"""Plain fp64 CPU oracle of the AsymSpec per-step decision path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product imports this module: only
``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import or run it.  It shares no code with the HIP library and
imports nothing from the package.

What it computes (AsymSpec, "Context-Asymmetric Speculative Decoding for
Agentic LLMs", arXiv 2608.26004):

* Sec. 3.2, Eq. 1   context-gain signal   delta_i = a_i - b_i  (logit space)
* Sec. 3.2, Eq. 2   delta-fused emission  d'_i = argmax(t_i + beta * delta_i)
* Sec. 3.3, Eq. 3   CDA gate  gamma_eff(i) = gamma * exp(-D_i),
                    D_i = JSD(softmax(a_i) || softmax(b_i))   (natural log,
                    so D_i <= ln 2 and gamma_eff in [gamma/2, gamma];
                    App. A derives the exponential form)
* Sec. 3.3, Eq. 4   greedy acceptance
                    softmax(t_i)[d_i] > gamma_eff(i) * softmax(b_i)[d_i]
* Alg. 1            accept the longest prefix of drafts, emit the fused argmax
                    at the first rejection and stop; if all K drafts pass,
                    append argmax(t_{K+1}) (the bonus row, unfused).

The paper defines the step for greedy decoding only (tau = 0; Sec. 3.3 ends by
saying the scheme is calibrated for greedy emission, and the Limitations
section leaves stochastic sampling to future work).  For tau > 0 this oracle
implements the reading that reduces to standard speculative sampling
(Leviathan et al. / Chen et al.) when delta = 0 and gamma = 1:

* fused target  p~ = softmax(f / tau), proposal q = softmax(a / tau);
* accept d_i iff u_i < min(1, p~(d_i) / (gamma_eff(i) * q(d_i)));
* at the first rejection emit a draw from the residual
  r(x) = max(0, p~(x) - q(x)) by inverse CDF with the caller uniform u_K;
* if all K drafts pass, draw the bonus from softmax(t_K / tau) with u_K.

Conventions fixed here (readings where the paper is silent or greedy-only):

* The fused logits f = t + beta*(a - b) are formed in IEEE fp32 in that order
  (no fused multiply-add): the argmax decisions of Eq. 2 are taken on these
  fp32 keys, lowest index on ties.  Everything downstream of f is fp64.
* A fused logit that is not a number (a = b = -inf: a token both drafter views
  mask) counts as masked (-inf).  Masked tokens carry zero probability.
* D_i is taken at temperature 1 for every row; terms with P = 0 or Q = 0
  contribute 0; the result is clamped to [0, ln 2].
* Each request's drafts/uniforms come in as inputs; this module draws no
  random numbers.

Variants the paper compares against (Sec. 6.2 mechanism ablation; App. B
"Models and hyperparameters" and the JSD-vs-KL table of App. G), selected by
``gate_mode`` and ``delta_mode``:

* gate FIXED   gamma_eff = gamma (standard speculative acceptance);
* gate KL      D_i = KL(softmax(a_i) || softmax(b_i)), natural log, not
               bounded (P = 0 terms are 0; P > 0 where Q = 0 gives +inf);
* gate LAMBDA  D_i = lambda * Delta_i(d_i), Delta = log softmax(a_i) -
               log softmax(b_i) taken at the draft token (the paper writes
               Delta as a vector; the gate needs its value at d_i);
* delta A      raw-augmented fusion, delta_i = a_i          (f = t + beta a);
* delta TB     SCD-style fusion, delta_i = t_i - b_i        (f = t + beta (t - b)).

``fuse_bonus`` fuses the bonus row too: Alg. 1 appends argmax(t_{K+1}), yet
the drafter logits of position K+1 are computed as well; with the flag the
bonus is taken from f_K = t_K + beta delta_K (greedy argmax, or a draw from
softmax(f_K / tau)) and rows K of a and b are read.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

LN2 = math.log(2.0)

GATE_CDA = 0      # gamma_eff = gamma * exp(-D)         (Sec. 3.3, Eq. 3)
GATE_FIXED = 1    # gamma_eff = gamma  (fixed-gamma baseline of App. B)
GATE_KL = 2       # gamma * exp(-KL(P || Q))            (App. G, JSD vs. KL)
GATE_LAMBDA = 3   # gamma * exp(-lambda * Delta(d))     (App. B, tuned-lambda foil)

DELTA_AB = 0      # delta = a - b   (Eq. 1, the paper's same-model source)
DELTA_A = 1       # delta = a       (raw-augmented, Sec. 6.2 ablation)
DELTA_TB = 2      # delta = t - b   (SCD-style, Sec. 6.2 ablation)


# --------------------------------------------------------------------------
# Storage decoding.  Inputs are bf16 (held as uint16 bit patterns) or fp32.
# --------------------------------------------------------------------------
def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> exact fp32 values (the bf16 value is the
    high half of an fp32 word)."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32)


def to_f32(x: np.ndarray) -> np.ndarray:
    """Stored logits -> fp32 (exact for both storage types)."""
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return bf16_bits_to_f32(x)
    if x.dtype == np.float32:
        return x
    raise TypeError(f"unsupported storage dtype {x.dtype}")


# --------------------------------------------------------------------------
# Sec. 3.2, Eq. 1-2: the fused logits.
# --------------------------------------------------------------------------
def fused_logits_f32(t32: np.ndarray, a32: np.ndarray, b32: np.ndarray,
                     beta: float, delta_mode: int = DELTA_AB) -> np.ndarray:
    """f = t + beta * delta, in fp32, in that order (Eq. 1 gives
    delta = a - b in logit space; Eq. 2 adds beta * delta to the verifier
    logits; the ablation's alternatives take delta = a or delta = t - b).
    NaN (only from -inf - (-inf), or inf * 0) is returned as -inf: the token
    is masked."""
    t32 = np.asarray(t32, np.float32)
    a32 = np.asarray(a32, np.float32)
    b32 = np.asarray(b32, np.float32)
    with np.errstate(invalid="ignore", over="ignore"):
        if delta_mode == DELTA_AB:
            delta = np.subtract(a32, b32, dtype=np.float32)
        elif delta_mode == DELTA_A:
            delta = a32
        elif delta_mode == DELTA_TB:
            delta = np.subtract(t32, b32, dtype=np.float32)
        else:
            raise ValueError(delta_mode)
        scaled = np.multiply(np.float32(beta), delta, dtype=np.float32)
        f = np.add(t32, scaled, dtype=np.float32)
    return np.where(np.isnan(f), np.float32(-np.inf), f).astype(np.float32)


def argmax_first(x: np.ndarray) -> int:
    """Index of the largest entry, the lowest index among equal maxima."""
    x = np.asarray(x)
    m = np.max(x)
    return int(np.flatnonzero(x == m)[0])


# --------------------------------------------------------------------------
# softmax / log-softmax (Eq. 3-4 use softmax of the logit rows).
# --------------------------------------------------------------------------
def log_softmax(x: np.ndarray, temperature: float = 1.0) -> np.ndarray:
    """log softmax(x / temperature) in fp64, written out: shift by the max,
    exponentiate, sum, take the log."""
    z = np.asarray(x, dtype=np.float64) / float(temperature)
    m = np.max(z)
    with np.errstate(divide="ignore"):
        lse = m + math.log(float(np.sum(np.exp(z - m))))
    return z - lse


def softmax(x: np.ndarray, temperature: float = 1.0) -> np.ndarray:
    return np.exp(log_softmax(x, temperature))


# --------------------------------------------------------------------------
# Sec. 3.3, Eq. 3: the divergence and the gate.
# --------------------------------------------------------------------------
def jsd(a: np.ndarray, b: np.ndarray) -> float:
    """D = JSD(softmax(a) || softmax(b)) with natural logarithms:
    D = 1/2 sum_x P log(P/M) + 1/2 sum_x Q log(Q/M),  M = (P + Q) / 2.
    Terms with P = 0 (resp. Q = 0) are 0.  Clamped to [0, ln 2] (the bound the
    paper states for D; App. A shows D is a mutual information of a binary
    channel)."""
    P = softmax(a)
    Q = softmax(b)
    M = 0.5 * (P + Q)
    tp = np.zeros_like(P)
    tq = np.zeros_like(Q)
    nzp = P > 0
    nzq = Q > 0
    tp[nzp] = P[nzp] * np.log(P[nzp] / M[nzp])
    tq[nzq] = Q[nzq] * np.log(Q[nzq] / M[nzq])
    d = 0.5 * float(np.sum(tp)) + 0.5 * float(np.sum(tq))
    return min(max(d, 0.0), LN2)


def kl(a: np.ndarray, b: np.ndarray) -> float:
    """KL(softmax(a) || softmax(b)) = sum_x P log(P/Q), natural log, not
    bounded.  Terms with P = 0 are 0; a token with P > 0 and Q = 0 makes it
    +inf."""
    P = softmax(a)
    Q = softmax(b)
    nz = P > 0
    if np.any(Q[nz] == 0):
        return math.inf
    return float(np.sum(P[nz] * np.log(P[nz] / Q[nz])))


def log_ratio_at(a: np.ndarray, b: np.ndarray, d: int) -> float:
    """Delta(d) = log softmax(a)[d] - log softmax(b)[d] (the tuned-lambda
    gate's per-position drafter log-probability difference, at the draft
    token)."""
    la = float(log_softmax(a)[d])
    lb = float(log_softmax(b)[d])
    if la == -math.inf and lb == -math.inf:
        return math.nan
    return la - lb


def gamma_eff(D: float, gamma: float, gate_mode: int = GATE_CDA) -> float:
    """Eq. 3: gamma_eff = gamma * exp(-D) (CDA, and the KL and lambda
    variants with their own D), or gamma (fixed-gamma gate)."""
    if gate_mode == GATE_FIXED:
        return float(gamma)
    return float(gamma) * math.exp(-float(D))


def divergence(a: np.ndarray, b: np.ndarray, d: int, gate_mode: int,
               lam: float) -> float:
    """The D of gamma_eff = gamma * exp(-D) for each gate (JSD for the CDA
    and fixed gates, where the fixed gate reports it without using it)."""
    if gate_mode == GATE_KL:
        return kl(a, b)
    if gate_mode == GATE_LAMBDA:
        return float(lam) * log_ratio_at(a, b, d)
    return jsd(a, b)


# --------------------------------------------------------------------------
# Per-row and per-request results.
# --------------------------------------------------------------------------
@dataclass
class RowResult:
    D: float = 0.0
    gamma_eff: float = 0.0
    accept: bool = False
    fused_logprob_draft: float = 0.0      # lp~_i(d_i)
    # distance of the decision from its threshold (for near-tie reporting)
    #   greedy: |exp(margin) - 1|,  sampling: |ratio - u|
    decision_gap: float = math.inf
    ratio: float = float("nan")           # sampling rows
    margin: float = float("nan")          # greedy rows, log of Eq. 4 ratio


@dataclass
class RequestResult:
    accept_len: int
    next_token: int
    fused_logprobs: np.ndarray            # [K+1]
    rows: list = field(default_factory=list)
    # distance of u_K from the nearest boundary of the inverse-CDF step that
    # picked next_token (sampling emissions), as a fraction of the mass
    emission_gap: float = math.inf
    emission_kind: str = ""               # "fused-argmax" | "residual" | "bonus-argmax" | "bonus-sample" | "residual-empty"

    def near_tie(self, tol: float = 1e-6) -> bool:
        """True when a decision that fixes (accept_len, next_token) lies
        within tol of its threshold: the acceptance of a row at or before the
        first rejection, or the inverse-CDF step that picked the token."""
        last = min(self.accept_len, len(self.rows) - 1)
        for i in range(0, last + 1):
            if i < len(self.rows) and self.rows[i].decision_gap < tol:
                return True
        return self.emission_gap < tol


def inverse_cdf(weights: np.ndarray, u: float) -> tuple[int, float]:
    """First index x with cumsum(w)[x] > u * sum(w) (inverse-CDF draw from the
    distribution proportional to w, w >= 0), and the distance of u from the
    two cumulative boundaries of that step, relative to the total."""
    w = np.asarray(weights, dtype=np.float64)
    c = np.cumsum(w)
    total = float(c[-1])
    target = float(u) * total
    x = int(np.searchsorted(c, target, side="right"))
    x = min(x, len(w) - 1)
    lo = float(c[x - 1]) if x > 0 else 0.0
    hi = float(c[x])
    gap = min(abs(target - lo), abs(hi - target)) / total
    return x, gap


def verify_request(t: np.ndarray, a: np.ndarray, b: np.ndarray,
                   draft_tokens: np.ndarray, draft_probs: np.ndarray | None,
                   uniforms: np.ndarray, temperature: float,
                   beta: float = 1.0, gamma: float = 0.5,
                   gate_mode: int = GATE_CDA, delta_mode: int = DELTA_AB,
                   lam: float = 0.1, fuse_bonus: bool = False) -> RequestResult:
    """One request of Alg. 1's decision step.

    t, a, b: stored logits [K+1][V] (uint16 bf16 bits or fp32).  Row K is the
    bonus position; rows K of a and b are not used (Alg. 1 appends
    argmax(t_{K+1}) unfused).  draft_tokens [K], draft_probs [K] or None,
    uniforms [K+1] (u_0..u_{K-1} acceptance, u_K emission draw),
    temperature <= 0 selects greedy decoding (the paper's setting)."""
    t32 = to_f32(t)
    a32 = to_f32(a)
    b32 = to_f32(b)
    Kp1, V = t32.shape
    K = Kp1 - 1
    tau = float(temperature)
    greedy = not (tau > 0.0)
    u = np.asarray(uniforms, dtype=np.float64)

    rows: list[RowResult] = []
    f_rows = []
    for i in range(K):
        d = int(draft_tokens[i])
        f = fused_logits_f32(t32[i], a32[i], b32[i], beta, delta_mode)  # Eq. 1-2
        f_rows.append(f)
        D = divergence(a32[i], b32[i], d, gate_mode, lam)        # Eq. 3
        ge = gamma_eff(D, gamma, gate_mode)                      # Eq. 3
        r = RowResult(D=D, gamma_eff=ge)
        # ln gamma_eff = ln gamma - D, kept in log form (D may be +inf)
        lge = math.log(gamma) if gate_mode == GATE_FIXED else math.log(gamma) - D
        if greedy:
            # Eq. 4 in log form: log p_t(d) - log p_b(d) - log gamma_eff > 0
            lpt = log_softmax(t32[i])[d]
            lpb = log_softmax(b32[i])[d]
            with np.errstate(invalid="ignore"):
                margin = float(lpt - lpb - lge)
            if math.isnan(margin):
                margin = -math.inf
            r.margin = margin
            r.accept = bool(margin > 0.0)
            r.decision_gap = abs(math.expm1(margin)) if np.isfinite(margin) else math.inf
            r.fused_logprob_draft = float(log_softmax(f)[d])
        else:
            lpf = log_softmax(f, tau)
            if draft_probs is not None:
                lq_d = math.log(float(draft_probs[i])) if draft_probs[i] > 0 else -math.inf
            else:
                lq_d = float(log_softmax(a32[i], tau)[d])
            lp_d = float(lpf[d])
            if lq_d == -math.inf and lp_d > -math.inf:
                ratio = 1.0
            elif lp_d == -math.inf:
                ratio = 0.0
            else:
                x = lp_d - lq_d - lge
                ratio = 0.0 if math.isnan(x) else min(1.0, math.exp(min(x, 0.0)))
            r.ratio = ratio
            r.accept = bool(u[i] < ratio)
            r.decision_gap = abs(ratio - float(u[i]))
            r.fused_logprob_draft = lp_d
        rows.append(r)

    # Alg. 1: the first rejection ends the step.
    accept_len = K
    for i in range(K):
        if not rows[i].accept:
            accept_len = i
            break

    flp = np.zeros(K + 1, dtype=np.float64)
    for i in range(K):
        flp[i] = rows[i].fused_logprob_draft

    emission_gap = math.inf
    if accept_len < K:
        j = accept_len
        f = f_rows[j]
        if greedy:
            nxt = argmax_first(f)                                # Eq. 2
            flp[K] = float(log_softmax(f)[nxt])
            kind = "fused-argmax"
        else:
            lpf = log_softmax(f, tau)
            lq = log_softmax(a32[j], tau)
            resid = np.maximum(0.0, np.exp(lpf) - np.exp(lq))
            if float(np.sum(resid)) > 0.0:
                nxt, emission_gap = inverse_cdf(resid, float(u[K]))
                kind = "residual"
            else:
                nxt = argmax_first(f)
                kind = "residual-empty"
            flp[K] = float(lpf[nxt])
    else:
        # Alg. 1 bonus: the verifier's last row, or its fused form
        tK = fused_logits_f32(t32[K], a32[K], b32[K], beta, delta_mode) if fuse_bonus else t32[K]
        if greedy:
            nxt = argmax_first(tK)
            flp[K] = float(log_softmax(tK)[nxt])
            kind = "bonus-argmax"
        else:
            lpt = log_softmax(tK, tau)
            nxt, emission_gap = inverse_cdf(np.exp(lpt), float(u[K]))
            flp[K] = float(lpt[nxt])
            kind = "bonus-sample"

    return RequestResult(accept_len=accept_len, next_token=int(nxt),
                         fused_logprobs=flp, rows=rows,
                         emission_gap=emission_gap, emission_kind=kind)


def fuse_verify(t, a, b, draft_tokens, draft_probs, uniforms, temperature,
                beta: float = 1.0, gamma: float = 0.5,
                gate_mode: int = GATE_CDA, requests=None,
                delta_mode: int = DELTA_AB, lam: float = 0.1, fuse_bonus: bool = False):
    """Batch form over requests: t, a, b [B][K+1][V]; draft_tokens [B][K];
    draft_probs [B][K] or None; uniforms [B][K+1]; temperature [B].
    ``requests`` restricts the work to a subset of request indices.
    Returns (accept_len [n], next_token [n], fused_logprobs [n][K+1],
    gate [n][K][2], list of RequestResult)."""
    B = t.shape[0]
    K = t.shape[1] - 1
    idx = list(range(B)) if requests is None else list(requests)
    n = len(idx)
    acc = np.zeros(n, np.int32)
    nxt = np.zeros(n, np.int32)
    flp = np.zeros((n, K + 1), np.float64)
    gate = np.zeros((n, K, 2), np.float64)
    res = []
    for k, bi in enumerate(idx):
        r = verify_request(t[bi], a[bi], b[bi], draft_tokens[bi],
                           None if draft_probs is None else draft_probs[bi],
                           uniforms[bi], float(temperature[bi]),
                           beta=beta, gamma=gamma, gate_mode=gate_mode,
                           delta_mode=delta_mode, lam=lam, fuse_bonus=fuse_bonus)
        acc[k] = r.accept_len
        nxt[k] = r.next_token
        flp[k] = r.fused_logprobs
        for i, row in enumerate(r.rows):
            gate[k, i, 0] = row.D
            gate[k, i, 1] = row.gamma_eff
        res.append(r)
    return acc, nxt, flp, gate, res


def fused_logprobs_full(t, a, b, temperature, beta: float = 1.0,
                        delta_mode: int = DELTA_AB, fuse_bonus: bool = False):
    """Every element's log-probability under its row's distribution, fp64
    [B][K+1][V]: rows i < K the fused target log softmax(f_i / tau) (Eq. 2,
    f in fp32 as in ``fused_logits_f32``, a NaN there counted as masked);
    row K the bonus distribution log softmax(t_K / tau) of Alg. 1, or of f_K
    with ``fuse_bonus``.  tau = 1 for a greedy request (tau <= 0), as for
    ``fused_logprobs``."""
    t32, a32, b32 = to_f32(t), to_f32(a), to_f32(b)
    B, Kp1, V = t32.shape
    K = Kp1 - 1
    out = np.empty((B, Kp1, V), dtype=np.float64)
    for bi in range(B):
        tau = float(temperature[bi])
        tau = tau if tau > 0.0 else 1.0
        for i in range(Kp1):
            if i < K or fuse_bonus:
                x = fused_logits_f32(t32[bi, i], a32[bi, i], b32[bi, i], beta, delta_mode)
            else:
                x = t32[bi, i]
            out[bi, i] = log_softmax(x, tau)
    return out


# --------------------------------------------------------------------------
# Sec. 6.4 and App. D: drafter and verifier from different model families.
# delta is computed in the drafter's vocabulary and carried to the
# verifier's through the string-identical tokens the two share; committed
# tokens are restricted to that set.  Reading: every distribution of the
# step is taken over the shared set, which is the same-vocabulary step on
# rows carried into the verifier's vocabulary with the unshared tokens masked
# in all three views.
# --------------------------------------------------------------------------
def map_to_verifier(t, a, b, vocab_map):
    """t [B][K+1][V] (verifier vocabulary), a and b [B][K+1][Vd] (drafter
    vocabulary), vocab_map [V] (drafter id of verifier token x, or -1).
    Returns (t', a', b') over the verifier vocabulary in the stored dtype:
    a'(x) = a(vocab_map[x]), b' likewise, and t' = t, where x is shared;
    -inf in all three where it is not."""
    vm = np.asarray(vocab_map, dtype=np.int64)
    Vd = a.shape[-1]
    shared = (vm >= 0) & (vm < Vd)
    j = np.where(shared, vm, 0)
    neg = np.uint16(0xFF80) if t.dtype == np.uint16 else np.float32(-np.inf)
    t2 = np.where(shared, t, neg).astype(t.dtype)
    a2 = np.where(shared, a[..., j], neg).astype(a.dtype)
    b2 = np.where(shared, b[..., j], neg).astype(b.dtype)
    return t2, a2, b2


def fuse_verify_xvocab(t, a, b, vocab_map, draft_tokens, draft_probs, uniforms,
                       temperature, **kw):
    """fuse_verify for a cross-family pair: the rows carried into the
    verifier's vocabulary first (``map_to_verifier``)."""
    t2, a2, b2 = map_to_verifier(t, a, b, vocab_map)
    return fuse_verify(t2, a2, b2, draft_tokens, draft_probs, uniforms, temperature, **kw)
