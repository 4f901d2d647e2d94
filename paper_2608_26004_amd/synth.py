"""Seeded synthetic inputs for the fused-verify step.

The paper's workloads (Qwen3 verifier/drafter logits on LongBench,
MultiChallenge, API-Bank, ...) need datasets and trained weights; these
generators stand in for them with logit rows shaped like real vocabularies
(32000, 128256, 151936, 256000 entries) and the structure the method reacts
to: a shared prior per position, verifier/drafter noise around it, and a
per-request divergence scale rho between the drafter's full view (a) and its
compressed view (b).

Every request draws from its own NumPy Philox stream,
``SeedSequence(seed).spawn(B)[b]``, so the output does not depend on how many
worker processes generate it.  Per request, in this order:

1. rho_b (and tau_b, fixed by the workload);
2. the prior z [K+1][V]: ``3 * N(0,1)``, or the Zipf-shaped
   ``-6*sqrt(ln rank) + N(0,1)`` with rank from a seeded permutation per row;
3. t = z + N(0,1), a = z + N(0,1), b = a + rho_b * N(0,1) (b is a bitwise copy
   of a when rho_b = 0);
4. rounding fp64 -> fp32 (round to nearest even) -> bf16 (round to nearest
   even) for bf16 workloads;
5. drafts from the *stored* a rows: for tau_b > 0 an inverse-CDF draw from
   softmax(a_i / tau_b) with one fp64 uniform, and draft_probs = fp32 of the
   drawn token's probability; for tau_b <= 0 the argmax and probability 1;
6. uniforms u [K+1] in [0, 1) as fp32 (u_0..u_{K-1} accept, u_K emission).

Step 5 models the drafter's own sampling, which happens upstream of the
decision step; nothing here computes any part of the decision step itself.
This module imports neither the oracle nor the HIP binding.
"""

from __future__ import annotations

import math
import os
from dataclasses import dataclass

import numpy as np

BF16 = "bf16"
FP32 = "fp32"


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    K: int
    V: int
    dtype: str           # "bf16" | "fp32"
    prior: str           # "gauss" | "zipf"
    rho: object          # float, ("uniform", lo, hi) or ("alternate", even, odd)
    tau: object          # float or ("alternate", even, odd)
    seed: int


# The five workloads of the benchmark suite.  Index = workload id.
WORKLOADS = [
    Workload("B1_K4_V32000_fp32", 1, 4, 32000, FP32, "gauss", 0.5, 1.0, 26004),
    Workload("B8_K5_V128256_bf16", 8, 5, 128256, BF16, "gauss", 1.0, 0.8, 26005),
    Workload("B32_K8_V151936_bf16_zipf", 32, 8, 151936, BF16, "zipf",
             ("uniform", 0.0, 2.0), 0.7, 26006),
    Workload("B128_K6_V151936_bf16", 128, 6, 151936, BF16, "gauss",
             ("alternate", 0.0, 3.0), 1.0, 26007),
    Workload("B512_K8_V256000_bf16_mixed", 512, 8, 256000, BF16, "gauss",
             ("uniform", 0.0, 2.0), ("alternate", 0.0, 1.0), 26008),
]


@dataclass
class Inputs:
    t: np.ndarray            # [B][K+1][V] uint16 (bf16 bits) or float32
    a: np.ndarray
    b: np.ndarray
    draft_tokens: np.ndarray  # [B][K] int32
    draft_probs: np.ndarray   # [B][K] float32
    uniforms: np.ndarray      # [B][K+1] float32
    temperature: np.ndarray   # [B] float32
    rho: np.ndarray           # [B] float64 (metadata)
    dtype: str

    @property
    def B(self):
        return self.t.shape[0]

    @property
    def K(self):
        return self.t.shape[1] - 1

    @property
    def V(self):
        return self.t.shape[2]

    def nbytes_read(self, fuse_bonus: bool = False) -> int:
        """Bytes the step reads from the logit streams: t rows 0..K, a and b
        rows 0..K-1; row K of a and b only when the bonus row is fused."""
        elem = 2 if self.dtype == BF16 else 4
        rows = 3 * (self.K + 1) if fuse_bonus else 3 * self.K + 1
        return self.B * rows * self.V * elem


def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp64 -> fp32 (RNE) -> bf16 bits (RNE).  Inputs are finite."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def stored_to_f64(x: np.ndarray) -> np.ndarray:
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


def _param(spec, b: int, rng: np.random.Generator) -> float:
    if isinstance(spec, (int, float)):
        return float(spec)
    kind = spec[0]
    if kind == "uniform":
        return float(rng.uniform(spec[1], spec[2]))
    if kind == "alternate":
        return float(spec[1] if b % 2 == 0 else spec[2])
    raise ValueError(spec)


def _draft(a_row: np.ndarray, tau: float, rng: np.random.Generator):
    """Drafter model: sample from softmax(a/tau) (tau > 0) or take the argmax."""
    if not tau > 0:
        return int(np.argmax(a_row)), 1.0
    z = (a_row - np.max(a_row)) / tau
    w = np.exp(z)
    c = np.cumsum(w)
    d = int(np.searchsorted(c, rng.random() * c[-1], side="right"))
    d = min(d, len(w) - 1)
    while w[d] == 0.0 and d > 0:      # never draft a zero-probability token
        d -= 1
    return d, float(w[d] / c[-1])


def _gen_request(wl_args, b, child_seed, mask_frac):
    """Generate request b; returns the stored rows and small arrays."""
    K, V, dtype, prior, rho_spec, tau_spec = wl_args
    rng = np.random.Generator(np.random.Philox(child_seed))
    rho = _param(rho_spec, b, rng)
    tau = _param(tau_spec, b, rng)
    if prior == "zipf":
        z = np.empty((K + 1, V))
        for i in range(K + 1):
            rank = rng.permutation(V).astype(np.float64) + 1.0
            z[i] = -6.0 * np.sqrt(np.log(rank)) + rng.standard_normal(V)
    else:
        z = 3.0 * rng.standard_normal((K + 1, V))
    t = z + rng.standard_normal((K + 1, V))
    a = z + rng.standard_normal((K + 1, V))
    nb = rng.standard_normal((K + 1, V))
    bb = a.copy() if rho == 0.0 else a + rho * nb
    if mask_frac > 0:
        mask = rng.random(V) < mask_frac
        t[:, mask] = -np.inf
        a[:, mask] = -np.inf
        bb[:, mask] = -np.inf
    if dtype == BF16:
        ts, as_, bs = (f64_to_bf16_bits(np.where(np.isinf(x), -3.0e38, x)) for x in (t, a, bb))
        if mask_frac > 0:
            for s in (ts, as_, bs):
                s[:, mask] = np.uint16(0xFF80)      # bf16 -inf
        a_stored = stored_to_f64(as_)
    else:
        ts, as_, bs = (x.astype(np.float32) for x in (t, a, bb))
        a_stored = as_.astype(np.float64)
    drafts = np.zeros(K, np.int32)
    dprobs = np.zeros(K, np.float32)
    for i in range(K):
        d, p = _draft(a_stored[i], tau, rng)
        drafts[i] = d
        dprobs[i] = np.float32(p)
    u = rng.random(K + 1, dtype=np.float32)
    return ts, as_, bs, drafts, dprobs, u, np.float32(tau), rho


def _worker(args):
    (shm_names, shape, np_dtype, wl_args, seeds, lo, hi, mask_frac) = args
    from multiprocessing import shared_memory
    shms = [shared_memory.SharedMemory(name=n) for n in shm_names]
    try:
        arrs = [np.ndarray(shape, dtype=np_dtype, buffer=s.buf) for s in shms]
        small = []
        for b in range(lo, hi):
            ts, as_, bs, d, p, u, tau, rho = _gen_request(wl_args, b, seeds[b - lo], mask_frac)
            arrs[0][b] = ts
            arrs[1][b] = as_
            arrs[2][b] = bs
            small.append((b, d, p, u, tau, rho))
        del arrs
        return small
    finally:
        for s in shms:
            s.close()


def generate(B: int, K: int, V: int, dtype: str = BF16, prior: str = "gauss",
             rho=1.0, tau=1.0, seed: int = 0, mask_frac: float = 0.0,
             workers: int | None = None) -> Inputs:
    """Seeded inputs for B requests of K drafts over a V-entry vocabulary."""
    if B < 1 or K < 0 or V < 1:
        raise ValueError("need B >= 1, K >= 0, V >= 1")
    children = np.random.SeedSequence(seed).spawn(B)
    wl_args = (K, V, dtype, prior, rho, tau)
    np_dtype = np.uint16 if dtype == BF16 else np.float32
    shape = (B, K + 1, V)
    total = B * (K + 1) * V
    if workers is None:
        workers = 1 if total * 3 < 64 * 2**20 else min(16, len(os.sched_getaffinity(0)))
    draft_tokens = np.zeros((B, K), np.int32)
    draft_probs = np.zeros((B, K), np.float32)
    uniforms = np.zeros((B, K + 1), np.float32)
    temperature = np.zeros(B, np.float32)
    rhos = np.zeros(B, np.float64)
    if workers <= 1 or B == 1:
        t = np.empty(shape, np_dtype)
        a = np.empty(shape, np_dtype)
        bb = np.empty(shape, np_dtype)
        for b in range(B):
            ts, as_, bs, d, p, u, tv, rv = _gen_request(wl_args, b, children[b], mask_frac)
            t[b], a[b], bb[b] = ts, as_, bs
            draft_tokens[b], draft_probs[b], uniforms[b] = d, p, u
            temperature[b], rhos[b] = tv, rv
        return Inputs(t, a, bb, draft_tokens, draft_probs, uniforms,
                      temperature, rhos, dtype)

    import multiprocessing as mp
    from multiprocessing import shared_memory
    nbytes = total * np.dtype(np_dtype).itemsize
    shms = [shared_memory.SharedMemory(create=True, size=max(nbytes, 1)) for _ in range(3)]
    try:
        per = math.ceil(B / workers)
        jobs = []
        for lo in range(0, B, per):
            hi = min(B, lo + per)
            jobs.append(([s.name for s in shms], shape, np_dtype, wl_args,
                         children[lo:hi], lo, hi, mask_frac))
        ctx = mp.get_context("spawn")
        with ctx.Pool(len(jobs)) as pool:
            for small in pool.map(_worker, jobs):
                for (b, d, p, u, tv, rv) in small:
                    draft_tokens[b], draft_probs[b], uniforms[b] = d, p, u
                    temperature[b], rhos[b] = tv, rv
        out = [np.ndarray(shape, dtype=np_dtype, buffer=s.buf).copy() for s in shms]
    finally:
        for s in shms:
            s.close()
            s.unlink()
    return Inputs(out[0], out[1], out[2], draft_tokens, draft_probs, uniforms,
                  temperature, rhos, dtype)


def workload_inputs(index: int, workers: int | None = None, **override) -> Inputs:
    """Inputs of benchmark workload ``index`` (0..4); keyword overrides
    (e.g. B=...) shrink it for quick checks."""
    wl = WORKLOADS[index]
    kw = dict(B=wl.B, K=wl.K, V=wl.V, dtype=wl.dtype, prior=wl.prior,
              rho=wl.rho, tau=wl.tau, seed=wl.seed)
    kw.update(override)
    return generate(workers=workers, **kw)


def workload_requests(index: int, lo: int, hi: int) -> Inputs:
    """Requests lo..hi-1 of benchmark workload ``index``, identical to the
    same requests of ``workload_inputs(index)`` (each request has its own
    seeded stream), so that a subset can be regenerated in another process."""
    wl = WORKLOADS[index]
    if not (0 <= lo < hi <= wl.B):
        raise ValueError("need 0 <= lo < hi <= B")
    children = np.random.SeedSequence(wl.seed).spawn(wl.B)
    wl_args = (wl.K, wl.V, wl.dtype, wl.prior, wl.rho, wl.tau)
    n = hi - lo
    np_dtype = np.uint16 if wl.dtype == BF16 else np.float32
    t = np.empty((n, wl.K + 1, wl.V), np_dtype)
    a = np.empty_like(t)
    bb = np.empty_like(t)
    d = np.zeros((n, wl.K), np.int32)
    p = np.zeros((n, wl.K), np.float32)
    u = np.zeros((n, wl.K + 1), np.float32)
    tau = np.zeros(n, np.float32)
    rho = np.zeros(n, np.float64)
    for k, b in enumerate(range(lo, hi)):
        t[k], a[k], bb[k], d[k], p[k], u[k], tau[k], rho[k] = _gen_request(wl_args, b, children[b], 0.0)
    return Inputs(t, a, bb, d, p, u, tau, rho, wl.dtype)


def replicate_for_mc(t_rows: np.ndarray, a_rows: np.ndarray, b_rows: np.ndarray,
                     tau: float, n: int, seed: int):
    """n copies of one request (rows [K+1][V], stored dtype) with fresh drafts
    d_i ~ softmax(a_i / tau) and fresh uniforms per copy, for Monte Carlo
    checks of the emitted law.  Returns (t, a, b, drafts, draft_probs,
    uniforms, temperature) batched over the copies."""
    rng = np.random.Generator(np.random.Philox(np.random.SeedSequence(seed)))
    Kp1, V = t_rows.shape
    K = Kp1 - 1
    a64 = stored_to_f64(a_rows)
    drafts = np.zeros((n, K), np.int32)
    dprobs = np.zeros((n, K), np.float32)
    for i in range(K):
        z = (a64[i] - np.max(a64[i])) / tau
        w = np.exp(z)
        c = np.cumsum(w)
        d = np.searchsorted(c, rng.random(n) * c[-1], side="right")
        d = np.minimum(d, V - 1)
        drafts[:, i] = d
        dprobs[:, i] = (w[d] / c[-1]).astype(np.float32)
    uniforms = rng.random((n, K + 1), dtype=np.float32)
    t = np.broadcast_to(t_rows, (n, Kp1, V)).copy()
    a = np.broadcast_to(a_rows, (n, Kp1, V)).copy()
    b = np.broadcast_to(b_rows, (n, Kp1, V)).copy()
    temperature = np.full(n, tau, np.float32)
    return t, a, b, drafts, dprobs, uniforms, temperature


def cross_vocab(inp: Inputs, Vd: int, n_shared: int, seed: int = 0):
    """A drafter of another model family for `inp` (App. D's setting):
    drafter rows over a vocabulary of Vd tokens that hold inp.a / inp.b at
    the drafter ids of n_shared verifier tokens (both chosen at random, a
    stand-in for the string-identical tokens of two tokenizers), the other
    drafter tokens filled with N(0, 3^2) noise, and the map [V] int32 (drafter
    id of each verifier token, -1 for the unshared ones).  Drafts that fall
    outside the shared set are moved to a shared token of the same request
    (the drafter commits shared tokens only).  Returns (a_d, b_d, vocab_map,
    draft_tokens)."""
    rng = np.random.default_rng(seed)
    B, Kp1, V = inp.t.shape
    n = min(V, Vd, n_shared)
    xs = np.sort(rng.choice(V, n, replace=False))
    vm = np.full(V, -1, np.int32)
    vm[xs] = rng.choice(Vd, n, replace=False).astype(np.int32)
    def noise():
        x = rng.normal(0.0, 3.0, (B, Kp1, Vd))
        return f64_to_bf16_bits(x) if inp.dtype == BF16 else x.astype(np.float32)
    ad, bd = noise(), noise()
    ad[..., vm[xs]] = inp.a[..., xs]
    bd[..., vm[xs]] = inp.b[..., xs]
    d = inp.draft_tokens.copy()
    bad = vm[d] < 0
    d[bad] = xs[rng.integers(0, n, int(bad.sum()))]
    return ad, bd, vm, d
