"""Multi-step speculative decoding over table-driven stand-in models.

The loop of Alg. 1 around the decision step: per step the drafter proposes
K tokens autoregressively from its full-context view, the three logit rows of
every position are produced (drafter full view a, drafter compressed view b,
verifier t; Alg. 1 runs the three forwards), ``fuse_verify`` decides, and the
accepted drafts plus the emitted token are committed.  It reports the two
acceptance diagnostics of the paper's acceptance table (App. F):

  AR   accepted drafts / drafts evaluated, where the drafts evaluated in a
       step are the accepted ones plus the first rejected one (Alg. 1 stops
       there; K when all are accepted);
  MAL  mean number of tokens committed per step, accept_len + 1, out of the
       K + 1 positions.

The "models" are stand-ins (no weights are available): three tables of R
logit rows each, indexed by a rolling hash of the context.  A shared prior z
per table row gives the views their agreement; t = z + N(0,1),
a = z + N(0,1), b = a + rho N(0,1) (b is a copy of a when rho = 0), stored in
the logit dtype.  Drafting happens on the host from the stored a rows (it
stands in for the drafter's own sampler, upstream of the decision step); the
rows of the K+1 positions are gathered from device copies of the tables, and
only hashes, drafts and uniforms cross PCIe.
"""

from __future__ import annotations

import argparse
import json
import time

import numpy as np

from . import synth

_MUL = 1000003
_MASK = 0x7FFFFFFF


def roll(h, tok):
    """Context hash after appending token(s) `tok` (int64 arrays or ints)."""
    return (np.asarray(h, dtype=np.int64) * _MUL + np.asarray(tok, dtype=np.int64) + 1) & _MASK


class TableModels:
    """Verifier / drafter stand-ins: R rows of V logits per view."""

    def __init__(self, V: int, R: int = 512, rho: float = 1.0, prior_scale: float = 3.0,
                 dtype: str = synth.BF16, seed: int = 0, device=None, identical: bool = False):
        rng = np.random.default_rng(seed)
        z = prior_scale * rng.standard_normal((R, V))
        t = z + rng.standard_normal((R, V))
        a = t.copy() if identical else z + rng.standard_normal((R, V))
        b = a.copy() if (identical or rho == 0.0) else a + rho * rng.standard_normal((R, V))
        if dtype == synth.BF16:
            self.host = [synth.f64_to_bf16_bits(x) for x in (t, a, b)]
        else:
            self.host = [x.astype(np.float32) for x in (t, a, b)]
        self.V, self.R, self.dtype = V, R, dtype
        self.dev = None
        if device is not None:
            import torch
            if dtype == synth.BF16:
                self.dev = [torch.from_numpy(x.view(np.int16)).to(device).view(torch.bfloat16)
                            for x in self.host]
            else:
                self.dev = [torch.from_numpy(x).to(device) for x in self.host]

    def row_index(self, h):
        return np.asarray(h, dtype=np.int64) % self.R

    def drafter_row_f64(self, h):
        return synth.stored_to_f64(self.host[1][int(self.row_index(h))])


def _draft_token(a_row: np.ndarray, tau: float, u: float):
    """The drafter's own choice from its full-view row: argmax (tau <= 0) or
    an inverse-CDF draw from softmax(a / tau) with uniform u; returns the
    token and its proposal probability."""
    if not tau > 0:
        return int(np.argmax(a_row)), 1.0
    z = (a_row - np.max(a_row)) / tau
    w = np.exp(z)
    c = np.cumsum(w)
    d = min(int(np.searchsorted(c, u * c[-1], side="right")), len(w) - 1)
    while w[d] == 0.0 and d > 0:
        d -= 1
    return d, float(w[d] / c[-1])


class SpecDecoder:
    """B independent requests decoded with K drafts per step.

    backend "hip": rows gathered on the GPU and the step runs through
    ``fuse_verify``.  backend "host": rows gathered as NumPy arrays and passed
    to ``step_fn(t, a, b, d, q, u, tau) -> (accept_len, next_token)`` (a
    checker; the product path is "hip")."""

    def __init__(self, models: TableModels, B: int, K: int, temperature, beta: float = 1.0,
                 gamma: float = 0.5, gate_mode: int = 0, seed: int = 0, backend: str = "hip",
                 step_fn=None, device=None, early_exit: int = 0, fuse_bonus: bool = False):
        self.m, self.B, self.K = models, B, K
        self.tau = np.broadcast_to(np.asarray(temperature, np.float32), (B,)).copy()
        self.beta, self.gamma, self.gate_mode = beta, gamma, gate_mode
        self.early_exit, self.fuse_bonus = early_exit, fuse_bonus
        self.call_seconds = []
        self.rng = np.random.default_rng(seed)
        self.h = roll(np.zeros(B, np.int64), np.arange(B))     # distinct start contexts
        self.tokens = [[] for _ in range(B)]
        self.backend, self.step_fn, self.device = backend, step_fn, device
        self.accepted = 0
        self.evaluated = 0
        self.committed = 0
        self.steps = 0
        self.log = []
        if backend == "hip":
            import torch
            import paper_2608_26004_amd as asp
            if models.dev is None:
                raise ValueError("the hip backend needs TableModels(device=...)")
            self._torch, self._asp = torch, asp
            self._ws = asp.Workspace(device)
            self._tau_dev = torch.from_numpy(self.tau).to(device)
        elif step_fn is None:
            raise ValueError("the host backend needs step_fn")

    def _draft(self):
        B, K = self.B, self.K
        d = np.zeros((B, K), np.int32)
        q = np.zeros((B, K), np.float32)
        hs = np.zeros((B, K + 1), np.int64)
        ud = self.rng.random((B, K))
        for b in range(B):
            h = self.h[b]
            for i in range(K):
                hs[b, i] = h
                tok, p = _draft_token(self.m.drafter_row_f64(h), float(self.tau[b]), float(ud[b, i]))
                d[b, i], q[b, i] = tok, np.float32(p)
                h = roll(h, tok)
            hs[b, K] = h
        return d, q, hs

    def step(self):
        B, K = self.B, self.K
        d, q, hs = self._draft()
        u = self.rng.random((B, K + 1), dtype=np.float32)
        idx = self.m.row_index(hs).reshape(-1)
        if self.backend == "hip":
            torch = self._torch
            ii = torch.from_numpy(idx).to(self.device)
            t, a, b = (x.index_select(0, ii).view(B, K + 1, self.m.V) for x in self.m.dev)
            dd, qq, uu = (torch.from_numpy(v).to(self.device) for v in (d, q, u))
            torch.cuda.synchronize(self.device)
            t0 = time.perf_counter()
            acc, nxt, _ = self._asp.fuse_verify(
                t, a, b, dd, qq, uu, self._tau_dev, beta=self.beta, gamma=self.gamma,
                gate_mode=self.gate_mode, workspace=self._ws, early_exit=self.early_exit,
                fuse_bonus=self.fuse_bonus)
            acc, nxt = acc.cpu().numpy(), nxt.cpu().numpy()
            self.call_seconds.append(time.perf_counter() - t0)
        else:
            t, a, b = (x[idx].reshape(B, K + 1, self.m.V) for x in self.m.host)
            acc, nxt = self.step_fn(t, a, b, d, q, u, self.tau)
            acc, nxt = np.asarray(acc), np.asarray(nxt)
        for r in range(B):
            j = int(acc[r])
            new = [int(x) for x in d[r, :j]] + [int(nxt[r])]
            self.tokens[r].extend(new)
            h = hs[r, j]
            self.h[r] = roll(h, int(nxt[r]))
            self.accepted += j
            self.evaluated += j + (1 if j < K else 0)
            self.committed += len(new)
        self.steps += 1
        self.log.append((acc.copy(), nxt.copy()))
        return acc, nxt

    def report(self):
        n = self.steps * self.B
        rep = {"steps": self.steps, "requests": self.B, "K": self.K,
               "AR": self.accepted / self.evaluated if self.evaluated else float("nan"),
               "MAL": self.committed / n if n else float("nan"),
               "tokens": self.committed}
        if self.backend == "hip" and len(self.call_seconds) > 1:
            # host-observed latency of the decision call (median, first call
            # excluded): argument checks, launch, the kernel, and the copy of
            # accept_len and next_token back
            rep["decision_call_us"] = 1e6 * float(np.median(self.call_seconds[1:]))
        return rep


def main(argv=None):
    ap = argparse.ArgumentParser(description="multi-step speculative decoding over stand-in models")
    ap.add_argument("--B", type=int, default=8)
    ap.add_argument("--K", type=int, default=2)
    ap.add_argument("--V", type=int, default=32000)
    ap.add_argument("--R", type=int, default=512)
    ap.add_argument("--rho", type=float, default=1.0)
    ap.add_argument("--tau", type=float, default=0.0)
    ap.add_argument("--beta", type=float, default=1.0)
    ap.add_argument("--gamma", type=float, default=0.5)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--dtype", choices=[synth.BF16, synth.FP32], default=synth.BF16)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--gate", choices=["cda", "fixed", "kl", "lambda"], default="cda")
    ap.add_argument("--early-exit", type=int, default=0)
    args = ap.parse_args(argv)
    import torch
    dev = torch.device("cuda")
    models = TableModels(args.V, R=args.R, rho=args.rho, dtype=args.dtype, seed=args.seed, device=dev)
    gm = {"cda": 0, "fixed": 1, "kl": 2, "lambda": 3}[args.gate]
    dec = SpecDecoder(models, args.B, args.K, args.tau, beta=args.beta, gamma=args.gamma,
                      gate_mode=gm, seed=args.seed + 1, device=dev, early_exit=args.early_exit)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        dec.step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    rep = dec.report()
    rep.update({"V": args.V, "tau": args.tau, "beta": args.beta, "gamma": args.gamma,
                "rho": args.rho, "gate": args.gate, "early_exit": args.early_exit, "wall_s": wall})
    print(json.dumps(rep))


if __name__ == "__main__":
    main()
