"""Shared helpers for the GPU parity tests: numpy inputs -> device tensors,
one call through the C ABI, and the comparison with the CPU oracle.

Parity protocol
  * accept_len and next_token bit-exact, except requests whose decisions lie
    within NEAR_TIE of a threshold in the oracle (|ratio - u| for sampling
    acceptance, |exp(margin) - 1| for Eq. 4, the distance of u_K from an
    inverse-CDF step boundary for sampled emissions); those are counted and
    reported separately;
  * fused_logprobs within LP_TOL absolute (entry K only for requests whose
    outcome matches);
  * gate (D, gamma_eff) within LP_TOL absolute below 1 and relative above
    (the KL gate's D is not bounded).
"""

import numpy as np

import oracle as O

NEAR_TIE = 1e-6
LP_TOL = 1e-5


def to_device(x, device="cuda"):
    import torch
    if x.dtype == np.uint16:
        return torch.from_numpy(x.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(x)).to(device)


def run_gpu(inp, beta=1.0, gamma=0.5, gate_mode=0, with_probs=True, want_gate=True,
            device="cuda", delta_mode=0, lam=0.1, fuse_bonus=False, want_full=False, vocab=None,
            early_exit=0):
    """vocab = (a_d, b_d, vocab_map): drafter rows in another vocabulary,
    passed in place of inp.a and inp.b."""
    import torch
    import paper_2608_26004_amd as asp
    t, a, b = (to_device(x, device) for x in (inp.t, inp.a, inp.b))
    vm = None
    if vocab is not None:
        a, b = (to_device(x, device) for x in vocab[:2])
        vm = to_device(np.asarray(vocab[2], np.int32), device)
    d = to_device(inp.draft_tokens.astype(np.int32), device)
    q = to_device(inp.draft_probs.astype(np.float32), device) if with_probs else None
    u = to_device(inp.uniforms.astype(np.float32), device)
    tau = to_device(inp.temperature.astype(np.float32), device)
    ws = asp.Workspace(t.device)
    out = asp.fuse_verify(t, a, b, d, q, u, tau, beta=beta, gamma=gamma,
                          gate_mode=gate_mode, return_gate=want_gate,
                          delta_mode=delta_mode, lam=lam, fuse_bonus=fuse_bonus,
                          return_full=want_full, vocab_map=vm, early_exit=early_exit,
                          workspace=ws)
    torch.cuda.synchronize()
    # every wait between the launch's workgroups ended in time
    n_to = ws.timeouts()
    assert n_to == 0, f"{n_to} timed-out waits"
    res = [x.cpu().numpy() for x in out]
    if not want_gate:
        res.insert(3, None)
    return res


def _oracle_chunk(job):
    w, lo, hi, kw = job
    from paper_2608_26004_amd import synth
    x = synth.workload_requests(w, lo, hi)
    return lo, O.fuse_verify(x.t, x.a, x.b, x.draft_tokens, x.draft_probs, x.uniforms,
                             x.temperature, **kw)


def oracle_workload(w, procs=16, **kw):
    """The oracle over every request of benchmark workload w, in a pool of
    `procs` spawned processes that each regenerate their share of the
    requests from the seeded per-request streams (no fork of a process that
    holds a GPU context).  Returns what oracle.fuse_verify returns."""
    import multiprocessing as mp
    from paper_2608_26004_amd import synth
    B = synth.WORKLOADS[w].B
    procs = max(1, min(procs, B))
    per = -(-B // procs)
    jobs = [(w, lo, min(B, lo + per), kw) for lo in range(0, B, per)]
    with mp.get_context("spawn").Pool(len(jobs)) as pool:
        parts = sorted(pool.map(_oracle_chunk, jobs), key=lambda r: r[0])
    outs = [p[1] for p in parts]
    return (np.concatenate([o[0] for o in outs]), np.concatenate([o[1] for o in outs]),
            np.concatenate([o[2] for o in outs]), np.concatenate([o[3] for o in outs]),
            [r for o in outs for r in o[4]])


def near_tie_budget(n_rows):
    """Near-ties allowed per config: more than 1e-4 of the rows signals a
    bug (at least one is allowed)."""
    return max(1, int(1e-4 * n_rows))


def compare(inp, gpu, beta=1.0, gamma=0.5, gate_mode=0, with_probs=True,
            requests=None, label="", delta_mode=0, lam=0.1, fuse_bonus=False, oracle_out=None):
    """Run the oracle on `requests` (all by default) and compare (or take the
    oracle's results over those requests from `oracle_out`).  Returns a dict
    report; raises AssertionError on a parity failure."""
    acc_g, nxt_g, flp_g, gate_g = gpu[:4]
    idx = list(range(inp.B)) if requests is None else list(requests)
    if oracle_out is None:
        oracle_out = O.fuse_verify(
            inp.t, inp.a, inp.b, inp.draft_tokens, inp.draft_probs if with_probs else None,
            inp.uniforms, inp.temperature, beta=beta, gamma=gamma, gate_mode=gate_mode,
            requests=idx, delta_mode=delta_mode, lam=lam, fuse_bonus=fuse_bonus)
    acc_o, nxt_o, flp_o, gate_o, res = oracle_out
    assert len(acc_o) == len(idx)
    K = inp.K
    near, bad = [], []
    max_lp = 0.0
    max_gate = 0.0
    for k, bi in enumerate(idx):
        same = acc_g[bi] == acc_o[k] and nxt_g[bi] == nxt_o[k]
        tie = res[k].near_tie(NEAR_TIE)
        if not same:
            (near if tie else bad).append((bi, int(acc_g[bi]), int(nxt_g[bi]),
                                           int(acc_o[k]), int(nxt_o[k])))
        hi = K + 1 if same else K
        if hi > 0:
            with np.errstate(invalid="ignore"):     # -inf - -inf where both are masked
                d = np.abs(flp_g[bi, :hi].astype(np.float64) - flp_o[k, :hi])
            finite = np.isfinite(flp_o[k, :hi])
            if np.any(finite != np.isfinite(flp_g[bi, :hi])):
                bad.append((bi, "non-finite mismatch", flp_g[bi, :hi].tolist(), flp_o[k, :hi].tolist()))
            elif finite.any():
                max_lp = max(max_lp, float(d[finite].max()))
        if gate_g is not None and K > 0:
            # absolute below 1, relative above (the KL gate's D is not
            # bounded); infinities must agree
            gg = gate_g[bi].astype(np.float64)
            go = gate_o[k]
            fin = np.isfinite(go)
            if np.any(fin != np.isfinite(gg)) or np.any(gg[~fin] != go[~fin]):
                bad.append((bi, "gate non-finite mismatch", gg.tolist(), go.tolist()))
            elif fin.any():
                err = np.abs(gg[fin] - go[fin]) / np.maximum(1.0, np.abs(go[fin]))
                max_gate = max(max_gate, float(err.max()))
    report = dict(label=label, requests=len(idx), mismatches=bad, near_ties=near,
                  max_lp_err=max_lp, max_gate_err=max_gate)
    assert not bad, f"{label}: parity failures {bad[:5]} (report {report})"
    assert max_lp <= LP_TOL, f"{label}: fused_logprobs error {max_lp}"
    assert max_gate <= LP_TOL, f"{label}: gate error {max_gate}"
    return report


def compare_full(inp, full_g, beta=1.0, delta_mode=0, fuse_bonus=False, requests=None, label=""):
    """Element-by-element check of the full log-probability rows against the
    oracle on `requests` (all by default): -inf exactly where the oracle has
    it, otherwise within LP_TOL absolute.  Returns the largest error."""
    idx = list(range(inp.B)) if requests is None else list(requests)
    full_o = O.fused_logprobs_full(inp.t[idx], inp.a[idx], inp.b[idx], inp.temperature[idx],
                                   beta=beta, delta_mode=delta_mode, fuse_bonus=fuse_bonus)
    g = full_g[idx].astype(np.float64)
    fin_o = np.isfinite(full_o)
    assert np.array_equal(fin_o, np.isfinite(g)), f"{label}: -inf pattern differs"
    assert (g[~fin_o] == full_o[~fin_o]).all(), f"{label}: non-finite values differ"
    err = float(np.abs(g[fin_o] - full_o[fin_o]).max()) if fin_o.any() else 0.0
    assert err <= LP_TOL, f"{label}: full log-prob error {err}"
    return err


def make_xvocab(inp, Vd, shared_frac, seed, unshared_drafts=False):
    """A cross-family version of `inp`: drafter rows in a vocabulary of Vd
    tokens holding inp.a / inp.b at the drafter ids of the shared verifier
    tokens (a random injection), drafter-only tokens filled with noise, and
    the map.  Returns (a_d, b_d, vocab_map, mapped) where `mapped` is `inp`
    with the rows the oracle sees (``map_to_verifier``)."""
    import copy
    rng = np.random.default_rng(seed)
    B, Kp1, V = inp.t.shape
    n_sh = min(V, Vd, max(1, int(round(shared_frac * V))))
    xs = np.sort(rng.choice(V, n_sh, replace=False))
    vm = np.full(V, -1, np.int32)
    vm[xs] = rng.choice(Vd, n_sh, replace=False)
    if inp.a.dtype == np.uint16:
        noise = lambda: f64_bits(rng.normal(0, 3, (B, Kp1, Vd)))
    else:
        noise = lambda: rng.normal(0, 3, (B, Kp1, Vd)).astype(np.float32)
    ad, bd = noise(), noise()
    ad[..., vm[xs]] = inp.a[..., xs]
    bd[..., vm[xs]] = inp.b[..., xs]
    mapped = copy.copy(inp)
    if not unshared_drafts and inp.K > 0:
        d = inp.draft_tokens.copy()
        bad = vm[d] < 0
        d[bad] = xs[rng.integers(0, n_sh, bad.sum())]
        mapped.draft_tokens = d
    mapped.t, mapped.a, mapped.b = O.map_to_verifier(inp.t, ad, bd, vm)
    return ad, bd, vm, mapped


def f64_bits(x):
    from paper_2608_26004_amd import synth
    return synth.f64_to_bf16_bits(x)
