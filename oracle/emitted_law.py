"""Closed-form law of (accept_len, next_token) for the sampling reading.

TEST INFRASTRUCTURE ONLY (see asymspec_ref.py).

With drafts drawn independently per row from the proposal q_i = softmax(a_i/tau)
and independent uniforms, the decision step of the sampling reading is a
product of per-row Bernoulli trials followed by one inverse-CDF draw:

  alpha_i = sum_d q_i(d) * min(1, p~_i(d) / (c_i * q_i(d)))      (c_i = gamma_eff)
  P(accept_len = j, next = x) = prod_{i<j} alpha_i * (1 - alpha_j) * r_j(x) / R_j
  P(accept_len = K, next = x) = prod_{i<K} alpha_i * softmax(t_K / tau)(x)

where r_j = max(0, p~_j - q_j) and R_j = sum_x r_j(x).  When c_i = 1 this is
the speculative-sampling construction of Leviathan et al. / Chen et al., for
which the law of the first emitted token equals p~_0 exactly; for c_i < 1 the
gate is lenient and the law differs (the paper says the scheme does not keep a
strict target distribution, Sec. 3.3).

The per-row quantities are recomputed here from the oracle's building blocks
(softmax of the fused logits, the JSD gate) so that this module shares the
oracle's definitions of p~, q and gamma_eff, but the probability arithmetic is
written independently of the sampler in asymspec_ref.verify_request.
"""

from __future__ import annotations

import math

import numpy as np

from .asymspec_ref import (GATE_CDA, fused_logits_f32, gamma_eff, jsd,
                           softmax, to_f32)


def row_quantities(t_row, a_row, b_row, tau, beta, gamma, gate_mode):
    """(p~, q, c) for one draft row."""
    t32, a32, b32 = to_f32(t_row), to_f32(a_row), to_f32(b_row)
    f = fused_logits_f32(t32, a32, b32, beta)
    p = softmax(f, tau)
    q = softmax(a32, tau)
    c = gamma_eff(jsd(a32, b32), gamma, gate_mode)
    return p, q, c


def acceptance_prob(p: np.ndarray, q: np.ndarray, c: float) -> float:
    """alpha = E_{d~q}[min(1, p(d) / (c q(d)))]."""
    s = 0.0
    for d in range(len(q)):
        if q[d] > 0:
            s += q[d] * min(1.0, p[d] / (c * q[d]))
    return s


def emitted_law(t, a, b, tau: float, beta: float = 1.0, gamma: float = 0.5,
                gate_mode: int = GATE_CDA) -> np.ndarray:
    """P[j, x] = P(accept_len = j, next_token = x), j = 0..K, for one request
    whose drafts are drawn from q_i (sampling reading, tau > 0).
    t, a, b: [K+1][V] stored logits."""
    if not tau > 0:
        raise ValueError("the law is random only for tau > 0")
    K = t.shape[0] - 1
    V = t.shape[1]
    P = np.zeros((K + 1, V))
    survive = 1.0
    for j in range(K):
        p, q, c = row_quantities(t[j], a[j], b[j], tau, beta, gamma, gate_mode)
        alpha = acceptance_prob(p, q, c)
        r = np.maximum(0.0, p - q)
        R = float(np.sum(r))
        if R > 0:
            P[j] = survive * (1.0 - alpha) * r / R
        else:
            # residual is empty only when p~ == q, and then alpha == 1
            P[j, int(np.argmax(fused_logits_f32(to_f32(t[j]), to_f32(a[j]),
                                                to_f32(b[j]), beta)))] = survive * (1.0 - alpha)
        survive *= alpha
    P[K] = survive * softmax(to_f32(t[K]), tau)
    return P


def first_token_law(t, a, b, tau: float, beta: float = 1.0, gamma: float = 0.5,
                    gate_mode: int = GATE_CDA) -> np.ndarray:
    """Law of the first token the step commits (the accepted d_0, or the
    emission at row 0 when d_0 is rejected)."""
    p, q, c = row_quantities(t[0], a[0], b[0], tau, beta, gamma, gate_mode)
    V = len(p)
    law = np.zeros(V)
    for x in range(V):
        if q[x] > 0:
            law[x] += q[x] * min(1.0, p[x] / (c * q[x]))
    alpha = float(np.sum(law))
    r = np.maximum(0.0, p - q)
    R = float(np.sum(r))
    if R > 0:
        law += (1.0 - alpha) * r / R
    return law


def total_variation(p: np.ndarray, q: np.ndarray) -> float:
    return 0.5 * float(np.sum(np.abs(np.asarray(p) - np.asarray(q))))


def chi_square_stat(counts: np.ndarray, probs: np.ndarray) -> tuple[float, int]:
    """Pearson statistic over cells with expected count >= 5 (the rest are
    pooled into one cell); returns (statistic, degrees of freedom)."""
    counts = np.asarray(counts, dtype=np.float64).ravel()
    probs = np.asarray(probs, dtype=np.float64).ravel()
    n = counts.sum()
    exp = probs * n
    big = exp >= 5
    obs_b, exp_b = counts[big], exp[big]
    obs_s, exp_s = counts[~big].sum(), exp[~big].sum()
    stat = float(np.sum((obs_b - exp_b) ** 2 / exp_b))
    cells = int(big.sum())
    if exp_s > 0:
        stat += (obs_s - exp_s) ** 2 / exp_s
        cells += 1
    elif obs_s > 0:
        stat = math.inf
    return stat, max(cells - 1, 1)
