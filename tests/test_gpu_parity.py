"""GPU parity of the HIP decision step against the CPU oracle, through the
C ABI, on the seeded workloads and on edge shapes."""

import numpy as np
import pytest

import oracle as O
from paper_2608_26004_amd import synth

from parity_util import compare, compare_full, near_tie_budget, oracle_workload, run_gpu

pytestmark = pytest.mark.gpu


def _note(report):
    print(f"[parity] {report['label']}: {report['requests']} requests, "
          f"near-ties {len(report['near_ties'])}, max lp err {report['max_lp_err']:.2e}, "
          f"max gate err {report['max_gate_err']:.2e}", flush=True)


@pytest.fixture(scope="module")
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_26004_amd as asp
    asp.load_library()
    return torch.device("cuda")


# ------------------------------------------------------------ small cases --
@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("tau", [0.0, 1.0, 0.7])
def test_small_mixed(gpu, dtype, tau):
    x = synth.generate(B=6, K=3, V=5000, dtype=dtype, rho=("uniform", 0.0, 2.0), tau=tau, seed=11)
    for mode in (0, 1):
        g = run_gpu(x, gate_mode=mode)
        _note(compare(x, g, gate_mode=mode, label=f"small {dtype} tau={tau} mode={mode}"))


@pytest.mark.parametrize("B", [20, 40, 70])
def test_pass2_parts(gpu, B):
    """Pass 2 runs in 8, 4, 2 or 1 items per chunk depending on how many fit
    on the chip (B x 8 chunks of V = 120000: 4, 2 and 1 parts here, 8 in the
    small cases; at least 2 when the gate output is asked for under a
    JSD-based gate), each publishing its own partials; the emission draws
    and the divergence must not depend on the split."""
    x = synth.generate(B=B, K=2, V=120000, dtype="bf16", rho=("uniform", 0.0, 2.0),
                       tau=("alternate", 0.0, 1.0), seed=700 + B)
    for mode in (0, 1):
        for want_gate in (True, False):
            g = run_gpu(x, gate_mode=mode, want_gate=want_gate)
            _note(compare(x, g, gate_mode=mode, label=f"pass-2 parts B={B} mode={mode} gate={want_gate}"))


def test_argmax_ties_across_waves_and_chunks(gpu):
    """Greedy rows whose fused maximum is attained twice, in the runs of two
    waves of one statistics item and in two chunks: the first index wins
    (Eq. 2), whatever the order in which the partials are combined.  a = b,
    so f = t exactly and the tie is exact in every precision."""
    B, K, V = 2, 1, 20000             # bf16: 2 chunks of 16384 tokens
    x = synth.generate(B=B, K=K, V=V, dtype="bf16", rho=("uniform", 0.0, 1.0), tau=0.0, seed=77)
    def bf(v):
        return np.uint16(np.float32(v).view(np.uint32) >> 16)
    x.b[:] = x.a
    # the max of t at two tokens per request: 1500 (wave 0's run of chunk 0)
    # and 4500 (wave 1's); 16000 (chunk 0) and 16390 (chunk 1)
    ties = {0: (1500, 4500), 1: (16000, 16390)}
    for r, (i1, i2) in ties.items():
        x.t[r, :, i1] = bf(100.0)
        x.t[r, :, i2] = bf(100.0)
        d = int(x.draft_tokens[r, 0])
        if d in (i1, i2):
            d = (d + 7) % V
            x.draft_tokens[r, 0] = d
        # a sure rejection of draft 0: low verifier, high drafter logit
        x.t[r, 0, d] = bf(-4.0)
        x.a[r, 0, d] = x.b[r, 0, d] = bf(4.0)
    g = run_gpu(x)
    r = compare(x, g, label="argmax ties across waves and chunks")
    assert not r["near_ties"] or all(t[2] == t[4] for t in r["near_ties"])
    for req, (i1, _) in ties.items():
        assert int(g[0][req]) == 0 and int(g[1][req]) == i1


@pytest.mark.parametrize("V", [1, 2, 3, 5, 8, 4095, 4097, 8193, 32000])
@pytest.mark.parametrize("K", [0, 1, 4])
def test_edge_shapes(gpu, V, K):
    for dtype in ("bf16", "fp32"):
        x = synth.generate(B=5, K=K, V=V, dtype=dtype, rho=("uniform", 0.0, 2.0),
                           tau=("alternate", 0.0, 1.0), seed=V * 10 + K)
        g = run_gpu(x)
        _note(compare(x, g, label=f"edge V={V} K={K} {dtype}"))


def test_masked_tokens_and_identical_views(gpu):
    x = synth.generate(B=8, K=3, V=3001, dtype="bf16", rho=("alternate", 0.0, 1.5),
                       tau=("alternate", 0.0, 0.9), seed=5, mask_frac=0.1)
    g = run_gpu(x)
    r = compare(x, g, label="masked")
    _note(r)
    # identical drafter views: D = 0 and gamma_eff = gamma exactly
    gate = g[3]
    for bi in range(0, 8, 2):
        assert np.all(gate[bi, :, 0] == 0.0) and np.all(gate[bi, :, 1] == np.float32(0.5))


def test_shifted_comp_view_gives_zero_divergence(gpu):
    x = synth.generate(B=4, K=3, V=20000, dtype="fp32", rho=0.0, tau=0.0, seed=9)
    x.b[:] = (x.a.astype(np.float64) + 2.0).astype(np.float32)
    g = run_gpu(x)
    _note(compare(x, g, label="shifted b"))
    assert np.abs(g[3][:, :, 0]).max() < 1e-6


@pytest.mark.parametrize("beta,gamma", [(0.0, 1.0), (2.0, 0.5), (1.0, 1.0), (0.5, 0.25)])
def test_beta_gamma_grid(gpu, beta, gamma):
    x = synth.generate(B=8, K=4, V=7000, dtype="bf16", rho=("uniform", 0.0, 2.0),
                       tau=("alternate", 0.0, 1.0), seed=int(beta * 10 + gamma * 100))
    for mode in (0, 1):
        g = run_gpu(x, beta=beta, gamma=gamma, gate_mode=mode)
        _note(compare(x, g, beta=beta, gamma=gamma, gate_mode=mode,
                      label=f"beta={beta} gamma={gamma} mode={mode}"))


def test_draft_probs_null(gpu):
    x = synth.generate(B=8, K=4, V=9000, dtype="bf16", rho=1.0, tau=0.8, seed=21)
    g = run_gpu(x, with_probs=False)
    _note(compare(x, g, with_probs=False, label="draft_probs NULL"))


def test_without_gate_output_matches(gpu):
    x = synth.generate(B=12, K=4, V=6000, dtype="bf16", rho=("uniform", 0.0, 2.0),
                       tau=("alternate", 0.0, 1.0), seed=3)
    g1 = run_gpu(x, want_gate=True)
    g2 = run_gpu(x, want_gate=False)
    assert np.array_equal(g1[0], g2[0]) and np.array_equal(g1[1], g2[1])
    assert np.array_equal(g1[2], g2[2])
    _note(compare(x, g2, label="no gate"))


def test_determinism(gpu):
    x = synth.generate(B=16, K=5, V=12000, dtype="bf16", rho=("uniform", 0.0, 2.0),
                       tau=("alternate", 0.0, 1.0), seed=8)
    g1 = run_gpu(x)
    g2 = run_gpu(x)
    for u, v in zip(g1, g2):
        assert np.array_equal(u, v)


# --------------------------------------------------------------- workloads --
@pytest.mark.parametrize("w", [0, 1, 2])
def test_workload_full(gpu, w):
    x = synth.workload_inputs(w)
    g = run_gpu(x)
    r = compare(x, g, label=f"workload {w} ({synth.WORKLOADS[w].name})")
    _note(r)
    assert len(r["near_ties"]) <= max(1, int(1e-4 * x.B * (x.K + 1)))


def test_workload_3_full(gpu):
    """The bench workload (B=128, K=6, V=151936 bf16), every request, with
    and without the gate output; two runs are bitwise identical."""
    x = synth.workload_inputs(3)
    oo = oracle_workload(3)
    runs = []
    for want_gate in (True, False, False):
        g = run_gpu(x, want_gate=want_gate)
        r = compare(x, g, label=f"workload 3 gate={want_gate}", oracle_out=oo)
        _note(r)
        assert len(r["near_ties"]) <= near_tie_budget(x.B * (x.K + 1))
        runs.append(g)
    for u, v in zip(runs[1][:3], runs[2][:3]):
        assert np.array_equal(u, v)


def test_workload_4_full(gpu):
    """Full-size launch (B=512, K=8, V=256000, half greedy, half sampling),
    every request against the oracle (run in a pool of processes)."""
    x = synth.workload_inputs(4)
    g = run_gpu(x)
    oo = oracle_workload(4)
    r = compare(x, g, label="workload 4", oracle_out=oo)
    _note(r)
    assert len(r["near_ties"]) <= near_tie_budget(x.B * (x.K + 1))


# --------------------------------------------- gate and fusion variants --
# App. B (fixed and tuned-lambda gates), App. G (KL gate), Sec. 6.2 ablation
# (delta = a, delta = t - b), each against the oracle.
VARIANTS = [(2, 0), (3, 0), (0, 1), (0, 2), (2, 2), (3, 1), (1, 2)]


@pytest.mark.parametrize("gate,delta", VARIANTS)
@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("tau", [0.0, 1.0, 0.7])
def test_variants_small(gpu, gate, delta, dtype, tau):
    x = synth.generate(B=6, K=3, V=5000, dtype=dtype, rho=("uniform", 0.0, 2.0), tau=tau,
                       seed=100 + 10 * gate + delta)
    for lam in ((0.1, -2.0) if gate == 3 else (0.1,)):
        g = run_gpu(x, gate_mode=gate, delta_mode=delta, lam=lam)
        _note(compare(x, g, gate_mode=gate, delta_mode=delta, lam=lam,
                      label=f"variant gate={gate} delta={delta} lam={lam} {dtype} tau={tau}"))


@pytest.mark.parametrize("gate,delta", VARIANTS)
def test_variants_edges_and_masks(gpu, gate, delta):
    for V, K in ((1, 1), (4097, 2), (8193, 4)):
        x = synth.generate(B=4, K=K, V=V, dtype="bf16", rho=("uniform", 0.0, 2.0),
                           tau=("alternate", 0.0, 1.0), seed=V + K + gate)
        g = run_gpu(x, gate_mode=gate, delta_mode=delta)
        _note(compare(x, g, gate_mode=gate, delta_mode=delta, label=f"variant edge V={V} K={K} g={gate} d={delta}"))
    x = synth.generate(B=4, K=3, V=3000, dtype="fp32", rho=("uniform", 0.0, 2.0),
                       tau=("alternate", 0.0, 1.0), seed=7 + gate)
    # tokens every view masks, and tokens only the verifier masks (inputs
    # with b = -inf under a finite a or t give f = +inf: outside the contract)
    x.a[:, :, 10:20] = -np.inf
    x.b[:, :, 10:20] = -np.inf
    x.t[:, :, 10:25] = -np.inf
    x.b[1] = x.a[1]                     # identical views: D = 0 exactly
    g = run_gpu(x, gate_mode=gate, delta_mode=delta)
    _note(compare(x, g, gate_mode=gate, delta_mode=delta, label=f"variant masks g={gate} d={delta}"))


@pytest.mark.parametrize("gate,delta", [(2, 0), (3, 0), (0, 1), (0, 2)])
def test_variants_workload_1(gpu, gate, delta):
    x = synth.workload_inputs(1)
    g = run_gpu(x, gate_mode=gate, delta_mode=delta)
    _note(compare(x, g, gate_mode=gate, delta_mode=delta, label=f"variant workload 1 g={gate} d={delta}"))


def test_kl_gate_single_pass_infinite_and_zero_divergence(gpu):
    """KL gate (App. G) from the statistics items alone: a request whose
    compressed view masks tokens the full view keeps has D = +inf and
    gamma_eff = 0 (delta = a keeps the fused logits finite), requests with
    identical views have D = 0 exactly, the rest match the oracle; greedy
    and sampling requests, bf16 and fp32."""
    for dtype in ("fp32", "bf16"):
        x = synth.generate(B=8, K=3, V=4099, dtype=dtype, rho=("alternate", 0.0, 1.5),
                           tau=("alternate", 0.0, 1.0), seed=2 if dtype == "fp32" else 3)
        neg = np.float32(-np.inf) if dtype == "fp32" else np.uint16(0xFF80)
        x.b[1, :, 100:110] = neg
        x.b[5, :, 4000:4099] = neg
        g = run_gpu(x, gate_mode=2, delta_mode=1)
        _note(compare(x, g, gate_mode=2, delta_mode=1, label=f"KL +inf {dtype}"))
        gate = g[3]
        for r in (1, 5):
            assert np.isinf(gate[r, :, 0]).all() and (gate[r, :, 1] == 0.0).all()
        for r in (0, 2, 4, 6):
            assert (gate[r, :, 0] == 0.0).all() and (gate[r, :, 1] == np.float32(0.5)).all()


# ------------------------------------------------------ fused bonus row --
def _reach_bonus(x, reqs):
    """Requests `reqs` get identical views and verifier on their draft rows
    (t = a = b), so Eq. 4 and its sampling form accept every draft (ratio
    1 / gamma_eff >= 1; for sampling this needs delta = 0 there, i.e. not
    delta = a) and the step ends at the bonus row; row K keeps its own a and
    b.  Their draft probabilities are dropped (q computed from a)."""
    K = x.K
    for r in reqs:
        x.a[r, :K] = x.t[r, :K]
        x.b[r, :K] = x.t[r, :K]
    return x


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("tau", [0.0, 1.0, 0.7])
@pytest.mark.parametrize("gate,delta", [(0, 0), (2, 0), (3, 2), (1, 2), (1, 1)])
def test_fuse_bonus_small(gpu, dtype, tau, gate, delta):
    x = synth.generate(B=8, K=3, V=5000, dtype=dtype, rho=("uniform", 0.0, 2.0), tau=tau,
                       seed=300 + 10 * gate + delta)
    _reach_bonus(x, range(6))
    g = run_gpu(x, gate_mode=gate, delta_mode=delta, with_probs=False, fuse_bonus=True)
    r = compare(x, g, gate_mode=gate, delta_mode=delta, with_probs=False, fuse_bonus=True,
                label=f"fuse_bonus {dtype} tau={tau} g={gate} d={delta}")
    _note(r)
    if delta != 1 or tau == 0.0:
        assert (g[0][:6] == 3).all()
    # the flag reaches the kernel: the unfused bonus differs on some request
    g0 = run_gpu(x, gate_mode=gate, delta_mode=delta, with_probs=False)
    _note(compare(x, g0, gate_mode=gate, delta_mode=delta, with_probs=False,
                  label=f"unfused bonus {dtype} tau={tau} g={gate} d={delta}"))
    bon = g[0][:6] == 3
    if bon.any():
        assert (g0[1][:6][bon] != g[1][:6][bon]).any() or (g0[2][:6, 3][bon] != g[2][:6, 3][bon]).any()


@pytest.mark.parametrize("V,K", [(1, 0), (3, 0), (4097, 0), (4097, 2), (8193, 1)])
def test_fuse_bonus_edges(gpu, V, K):
    x = synth.generate(B=5, K=K, V=V, dtype="bf16", rho=("uniform", 0.0, 2.0),
                       tau=("alternate", 0.0, 1.0), seed=V + 7 * K)
    _reach_bonus(x, range(4))
    g = run_gpu(x, with_probs=False, fuse_bonus=True)
    _note(compare(x, g, with_probs=False, fuse_bonus=True, label=f"fuse_bonus edge V={V} K={K}"))


def test_fuse_bonus_masks(gpu):
    x = synth.generate(B=6, K=2, V=3000, dtype="fp32", rho=("uniform", 0.0, 2.0),
                       tau=("alternate", 0.0, 1.0), seed=77)
    _reach_bonus(x, range(6))
    # tokens every view masks (f is NaN there: masked), tokens only the
    # verifier masks, and a request whose bonus views agree (f_K = t_K)
    x.a[:, :, 10:20] = -np.inf
    x.b[:, :, 10:20] = -np.inf
    x.t[:, :, 10:25] = -np.inf
    x.b[2, 2] = x.a[2, 2]
    g = run_gpu(x, with_probs=False, fuse_bonus=True)
    _note(compare(x, g, with_probs=False, fuse_bonus=True, label="fuse_bonus masks"))


def test_fuse_bonus_workload_1(gpu):
    x = synth.workload_inputs(1)
    _reach_bonus(x, range(0, x.B, 2))
    g = run_gpu(x, with_probs=False, fuse_bonus=True)
    _note(compare(x, g, with_probs=False, fuse_bonus=True, label="fuse_bonus workload 1"))


# --------------------------------------------- full log-probability rows --
@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("tau", [0.0, 1.0, 0.7])
@pytest.mark.parametrize("delta,fb", [(0, False), (0, True), (1, False), (2, True)])
def test_full_logprobs_small(gpu, dtype, tau, delta, fb):
    x = synth.generate(B=5, K=3, V=5000, dtype=dtype, rho=("alternate", 0.0, 2.0), tau=tau,
                       seed=400 + delta)
    g = run_gpu(x, delta_mode=delta, fuse_bonus=fb, want_full=True)
    # the decision outputs are those of the call without the full rows
    g0 = run_gpu(x, delta_mode=delta, fuse_bonus=fb)
    for u, v in zip(g[:4], g0[:4]):
        assert np.array_equal(u, v)
    _note(compare(x, g, delta_mode=delta, fuse_bonus=fb, label=f"full {dtype} tau={tau} d={delta} fb={fb}"))
    err = compare_full(x, g[4], delta_mode=delta, fuse_bonus=fb, label=f"full {dtype} tau={tau}")
    print(f"[full] {dtype} tau={tau} delta={delta} fb={fb}: max abs err {err:.2e}")


@pytest.mark.parametrize("V,K", [(1, 0), (1, 2), (3, 1), (4097, 0), (4097, 3), (16385, 2)])
def test_full_logprobs_edges(gpu, V, K):
    x = synth.generate(B=3, K=K, V=V, dtype="bf16", rho=("uniform", 0.0, 2.0),
                       tau=("alternate", 0.0, 1.0), seed=V + K)
    for fb in (False, True):
        g = run_gpu(x, fuse_bonus=fb, want_full=True)
        compare_full(x, g[4], fuse_bonus=fb, label=f"full edge V={V} K={K} fb={fb}")


def test_full_logprobs_masks_and_beta(gpu):
    x = synth.generate(B=4, K=2, V=3000, dtype="fp32", rho=("uniform", 0.0, 2.0),
                       tau=("alternate", 0.0, 0.8), seed=91)
    x.a[:, :, 10:20] = -np.inf
    x.b[:, :, 10:20] = -np.inf
    x.t[:, :, 10:25] = -np.inf
    x.b[1] = x.a[1]
    for beta in (1.0, 0.35):
        g = run_gpu(x, beta=beta, want_full=True)
        compare_full(x, g[4], beta=beta, label=f"full masks beta={beta}")


def test_full_logprobs_workload_1(gpu):
    x = synth.workload_inputs(1)
    g = run_gpu(x, want_full=True)
    err = compare_full(x, g[4], requests=[0, 3, 7], label="full workload 1")
    print(f"[full] workload 1: max abs err {err:.2e}")


# ------------------------------------------- cross-family vocabularies --
# Sec. 6.4 / App. D: the drafter in its own vocabulary, reached through the
# map; the oracle sees the rows carried into the verifier's vocabulary.
def _run_xv(x, Vd, frac, seed, **kw):
    from parity_util import make_xvocab
    ad, bd, vm, mx = make_xvocab(x, Vd, frac, seed, unshared_drafts=kw.pop("unshared_drafts", False))
    g = run_gpu(mx, vocab=(ad, bd, vm), **kw)
    return g, mx


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("tau", [0.0, 1.0, 0.7])
@pytest.mark.parametrize("Vd,frac", [(4000, 0.7), (7000, 0.95), (5000, 1.0)])
def test_xvocab_small(gpu, dtype, tau, Vd, frac):
    x = synth.generate(B=5, K=3, V=5000, dtype=dtype, rho=("alternate", 0.0, 2.0), tau=tau,
                       seed=500 + Vd % 97)
    g, mx = _run_xv(x, Vd, frac, seed=Vd, want_full=True)
    _note(compare(mx, g, label=f"xvocab {dtype} tau={tau} Vd={Vd} frac={frac}"))
    compare_full(mx, g[4], label=f"xvocab full {dtype} tau={tau}")
    vm = np.asarray(_xv_map(mx))
    assert (vm[g[1]] >= 0).all()          # commits stay in the shared set


def _xv_map(mx):
    # the shared set as the oracle sees it: finite somewhere in t'
    fin = np.isfinite(synth.stored_to_f64(mx.t)).any(axis=(0, 1))
    return np.where(fin, 0, -1)


@pytest.mark.parametrize("gate,delta,fb", [(0, 0, True), (2, 0, False), (3, 2, False), (1, 1, True)])
def test_xvocab_variants(gpu, gate, delta, fb):
    x = synth.generate(B=6, K=2, V=3001, dtype="bf16", rho=("uniform", 0.0, 2.0),
                       tau=("alternate", 0.0, 1.0), seed=600 + gate)
    g, mx = _run_xv(x, 2500, 0.6, seed=gate, gate_mode=gate, delta_mode=delta, fuse_bonus=fb)
    _note(compare(mx, g, gate_mode=gate, delta_mode=delta, fuse_bonus=fb,
                  label=f"xvocab g={gate} d={delta} fb={fb}"))


@pytest.mark.parametrize("V,K,Vd", [(1, 1, 3), (7, 0, 5), (4097, 2, 300), (8193, 1, 9000)])
def test_xvocab_edges(gpu, V, K, Vd):
    x = synth.generate(B=3, K=K, V=V, dtype="bf16", rho=("uniform", 0.0, 2.0),
                       tau=("alternate", 0.0, 1.0), seed=V + Vd)
    g, mx = _run_xv(x, Vd, 0.8, seed=K, unshared_drafts=True, fuse_bonus=True, want_full=True)
    _note(compare(mx, g, fuse_bonus=True, label=f"xvocab edge V={V} K={K} Vd={Vd}"))
    compare_full(mx, g[4], fuse_bonus=True, label=f"xvocab edge full V={V}")


def test_xvocab_workload_1(gpu):
    x = synth.workload_inputs(1)
    g, mx = _run_xv(x, 120000, 0.85, seed=3)
    _note(compare(mx, g, label="xvocab workload 1"))


# ----------------------------------------------------------- early exit --
def _check_early_exit(x, ee, **kw):
    """Early exit against the full read of the same call (same kernels on
    the rows both read, so bitwise) and against the oracle: accept_len,
    next_token and fused_logprobs[K] agree; a draft row's outputs are NaN
    only after the first rejection (Alg. 1), otherwise they agree."""
    g0 = run_gpu(x, **kw)
    g = run_gpu(x, early_exit=ee, **kw)
    _note(compare(x, g0, label=f"early exit reference {kw}", **kw))
    acc0, nxt0, flp0, gate0 = g0[:4]
    acc, nxt, flp, gate = g[:4]
    assert np.array_equal(acc, acc0) and np.array_equal(nxt, nxt0)
    assert np.array_equal(flp[:, x.K], flp0[:, x.K], equal_nan=True)
    skipped = 0
    for r in range(x.B):
        for i in range(x.K):
            if np.isnan(flp[r, i]) and not np.isnan(flp0[r, i]):
                assert i > acc[r] and i >= ee, (r, i, acc[r])
                assert np.isnan(gate[r, i]).all()
                skipped += 1
            else:
                assert flp[r, i] == flp0[r, i] or (np.isnan(flp[r, i]) and np.isnan(flp0[r, i]))
                assert np.array_equal(gate[r, i], gate0[r, i], equal_nan=True)
    return skipped


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("tau", [0.0, 1.0, 0.7])
@pytest.mark.parametrize("ee", [1, 2, 4])
def test_early_exit_small(gpu, dtype, tau, ee):
    x = synth.generate(B=16, K=6, V=3000, dtype=dtype, rho=("alternate", 0.0, 2.0), tau=tau,
                       seed=700 + ee)
    n = _check_early_exit(x, ee)
    print(f"[early exit] {dtype} tau={tau} ee={ee}: {n} draft rows not read")


@pytest.mark.parametrize("gate,delta,fb", [(1, 0, True), (2, 0, False), (3, 2, True), (0, 1, False)])
def test_early_exit_variants(gpu, gate, delta, fb):
    x = synth.generate(B=12, K=5, V=4097, dtype="bf16", rho=("uniform", 0.0, 2.0),
                       tau=("alternate", 0.0, 1.0), seed=800 + gate)
    _check_early_exit(x, 2, gate_mode=gate, delta_mode=delta, fuse_bonus=fb)


@pytest.mark.parametrize("V,K,ee", [(1, 2, 1), (7, 1, 1), (8193, 3, 2), (5000, 2, 2), (300, 4, 9)])
def test_early_exit_edges(gpu, V, K, ee):
    x = synth.generate(B=6, K=K, V=V, dtype="bf16", rho=("uniform", 0.0, 2.0),
                       tau=("alternate", 0.0, 1.0), seed=V + K)
    _check_early_exit(x, ee)


def test_early_exit_xvocab(gpu):
    from parity_util import make_xvocab
    x = synth.generate(B=8, K=4, V=3000, dtype="bf16", rho=("uniform", 0.0, 2.0),
                       tau=("alternate", 0.0, 1.0), seed=901)
    ad, bd, vm, mx = make_xvocab(x, 2600, 0.8, seed=5)
    g0 = run_gpu(mx, vocab=(ad, bd, vm))
    g = run_gpu(mx, vocab=(ad, bd, vm), early_exit=2)
    _note(compare(mx, g0, label="early exit xvocab reference"))
    assert np.array_equal(g[0], g0[0]) and np.array_equal(g[1], g0[1])


def test_early_exit_workload_3_full(gpu):
    """The bench workload with early exit after two rows, every request:
    accept_len, next_token and fused_logprobs[K] against the oracle, the
    per-draft outputs on every row read (rows up to the first rejection)."""
    x = synth.workload_inputs(3)
    g = run_gpu(x, early_exit=2)
    acc, nxt, flp = g[0], g[1], g[2]
    acc_o, nxt_o, flp_o, _, res = oracle_workload(3)
    near = 0
    for bi in range(x.B):
        if (acc[bi], nxt[bi]) != (acc_o[bi], nxt_o[bi]):
            assert res[bi].near_tie(1e-6), (bi, acc[bi], nxt[bi], acc_o[bi], nxt_o[bi])
            near += 1
            continue
        assert abs(flp[bi, x.K] - flp_o[bi, x.K]) < 1e-5
        for i in range(min(acc[bi] + 1, x.K)):
            assert abs(flp[bi, i] - flp_o[bi, i]) < 1e-5
    assert near <= near_tie_budget(x.B * (x.K + 1))
    print(f"[early exit] workload 3: {int(np.isnan(flp[:, :x.K]).sum())} draft rows not read of "
          f"{x.B * x.K}, near-ties {near}")


# ------------------------------------------------------- maximum sizes --
def test_max_drafts(gpu):
    """K = 63: 64 rows per request, the most one wave's request-level logic
    holds."""
    x = synth.generate(B=2, K=63, V=1000, dtype="bf16", rho=("uniform", 0.0, 0.3),
                       tau=("alternate", 0.0, 1.0), seed=63)
    for ee in (0, 5):
        g = run_gpu(x, early_exit=ee)
        if ee == 0:
            _note(compare(x, g, label="K=63"))
        else:
            g0 = run_gpu(x)
            assert np.array_equal(g[0], g0[0]) and np.array_equal(g[1], g0[1])


@pytest.mark.parametrize("dtype,V", [("bf16", 4194297), ("fp32", 2097149)])
def test_max_vocabulary(gpu, dtype, V):
    """The longest rows the workspace layout takes: 256 chunks per row, so
    the decide item combines one row per group of 256 threads."""
    x = synth.generate(B=1, K=2, V=V, dtype=dtype, rho=1.0, tau=("alternate", 1.0, 0.0), seed=V % 1000)
    g = run_gpu(x, want_full=True)
    _note(compare(x, g, label=f"max V {dtype}"))
    compare_full(x, g[4], label=f"max V full {dtype}")


def test_many_requests(gpu):
    """A long item list: 3000 requests of tiny rows; the oracle checks a
    sample spread over the list (its start, middle and end)."""
    x = synth.generate(B=3000, K=1, V=64, dtype="fp32", rho=("uniform", 0.0, 2.0),
                       tau=("alternate", 0.0, 1.0), seed=3000)
    g = run_gpu(x)
    sample = list(range(0, 20)) + list(range(1490, 1510)) + list(range(2980, 3000))
    _note(compare(x, g, requests=sample, label="B=3000"))


# ------------------------------------------- the emitted law, sampled --
def _mc_rows(seed, K, V, equal_ab=False):
    rng = np.random.default_rng(seed)
    rows = lambda: (1.2 * rng.standard_normal((K + 1, V))).astype(np.float32)
    t, a = rows(), rows()
    b = a.copy() if equal_ab else rows()
    return t, a, b


def _mc_gpu(t, a, b, tau, n, seed, **kw):
    x = synth.Inputs(*synth.replicate_for_mc(t, a, b, tau, n, seed=seed), rho=np.zeros(n),
                     dtype="fp32")
    g = run_gpu(x, want_gate=False, **kw)
    return x, g[0], g[1]


@pytest.mark.parametrize("gamma,mode", [(0.5, 0), (0.7, 0), (1.0, 0), (0.5, 1)])
def test_emitted_law_monte_carlo(gpu, gamma, mode):
    """2^20 copies of one request in one launch, each with its own drafts
    (from q) and uniforms: the histogram of (accept_len, next_token) against
    the closed-form law of the sampling reading (oracle/emitted_law.py, an
    enumeration, not the oracle's sampler)."""
    import scipy.stats as sst
    K, V, tau = 2, 5, 0.9
    t, a, b = _mc_rows(31 + mode, K, V)
    x, acc, nxt = _mc_gpu(t, a, b, tau, 1 << 20, seed=5 + mode, gamma=gamma, gate_mode=mode)
    counts = np.zeros((K + 1, V))
    np.add.at(counts, (acc, nxt), 1)
    P = O.emitted_law(t, a, b, tau, gamma=gamma, gate_mode=mode)
    stat, dof = O.chi_square_stat(counts, P)
    p = sst.chi2.sf(stat, dof)
    n = counts.sum()
    z = np.abs(counts - n * P) / np.sqrt(np.maximum(n * P * (1 - P), 1e-12))
    print(f"[mc] gamma={gamma} mode={mode}: chi2 {stat:.1f} on {dof} dof, p {p:.3f}, max |z| {z.max():.2f}")
    assert p > 1e-3 and z.max() < 5.0


def test_speculative_sampling_theorem_on_gpu(gpu):
    """delta = 0 (a = b) and gamma = 1: the step is speculative sampling, so
    the first committed token follows softmax(t_0 / tau) exactly
    (Leviathan et al., Chen et al.), checked by chi-square over 2^20 copies."""
    import scipy.stats as sst
    import scipy.special as sps
    K, V, tau = 3, 6, 0.8
    t, a, b = _mc_rows(41, K, V, equal_ab=True)
    x, acc, nxt = _mc_gpu(t, a, b, tau, 1 << 20, seed=9, gamma=1.0)
    first = np.where(acc >= 1, x.draft_tokens[:, 0], nxt)
    counts = np.bincount(first, minlength=V).astype(np.float64)
    P = sps.softmax(t[0].astype(np.float64) / tau)
    stat, dof = O.chi_square_stat(counts, P)
    p = sst.chi2.sf(stat, dof)
    print(f"[mc] SD theorem: chi2 {stat:.1f} on {dof} dof, p {p:.3f}")
    assert p > 1e-3


def test_workload_3_invariants(gpu):
    """Properties that hold at any size, on the full bench workload: every
    full log-probability row normalises (Eq. 2 fused target), gamma_eff lies
    in [gamma/2, gamma] (Sec. 3.3), and the requests whose drafter views are
    bitwise equal (even b) have D = 0 and gamma_eff = gamma exactly."""
    import scipy.special as sps
    x = synth.workload_inputs(3)
    g = run_gpu(x, want_full=True)
    acc, nxt, flp, gate, full = g
    lse = sps.logsumexp(full.astype(np.float64), axis=-1)
    assert np.abs(lse).max() < 1e-5, np.abs(lse).max()
    ge = gate[..., 1]
    assert (ge >= 0.25 - 1e-7).all() and (ge <= 0.5 + 1e-7).all()
    even = np.arange(x.B) % 2 == 0
    assert (gate[even, :, 0] == 0.0).all() and (gate[even, :, 1] == np.float32(0.5)).all()
    assert (gate[~even, :, 0] > 0.0).all()


# ------------------------------------------------- a C caller, no Python --
def test_c_abi_example_program(gpu, tmp_path):
    """The example program calls the C ABI directly (hipMalloc, upload,
    asymspec_fuse_verify on its own stream, synchronise); its outputs match
    the oracle."""
    import os
    import subprocess
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    exe = os.path.join(root, "paper_2608_26004_amd", "examples", "fuse_verify_c")
    if not os.path.exists(exe):
        pytest.fail("the example program is not built (run __graft_entry__.build())")
    x = synth.generate(B=6, K=3, V=5003, dtype="bf16", rho=("uniform", 0.0, 2.0),
                       tau=("alternate", 0.0, 1.0), seed=2024)
    inp, out = tmp_path / "in.bin", tmp_path / "out.bin"
    with open(inp, "wb") as f:
        np.array([x.B, x.K, x.V, 0], np.int32).tofile(f)
        for arr in (x.t, x.a, x.b):
            np.ascontiguousarray(arr).tofile(f)
        x.draft_tokens.astype(np.int32).tofile(f)
        x.draft_probs.astype(np.float32).tofile(f)
        x.uniforms.astype(np.float32).tofile(f)
        x.temperature.astype(np.float32).tofile(f)
    r = subprocess.run([exe, str(inp), str(out)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    raw = np.fromfile(out, np.uint8)
    B, K = x.B, x.K
    acc = raw[:4 * B].view(np.int32)
    nxt = raw[4 * B:8 * B].view(np.int32)
    flp = raw[8 * B:8 * B + 4 * B * (K + 1)].view(np.float32).reshape(B, K + 1)
    gate = raw[8 * B + 4 * B * (K + 1):].view(np.float32).reshape(B, K, 2)
    _note(compare(x, [acc, nxt, flp, gate], label="C example"))


def test_xvocab_duplicate_map_entries(gpu):
    """Two verifier tokens naming the same drafter id (not a string-identical
    alignment, but a valid map): both take that drafter token's logits; the
    drafter-order path is not usable then and the verifier-order gathers
    give the oracle's result."""
    from parity_util import make_xvocab
    x = synth.generate(B=5, K=3, V=3000, dtype="bf16", rho=("uniform", 0.0, 2.0), tau=1.0, seed=17)
    ad, bd, vm, mx = make_xvocab(x, 2500, 0.8, seed=2)
    shared = np.nonzero(vm >= 0)[0]
    vm = vm.copy()
    vm[shared[1::7]] = vm[shared[0::7][:len(shared[1::7])]]     # duplicates
    mx.t, mx.a, mx.b = O.map_to_verifier(x.t, ad, bd, vm)
    g = run_gpu(mx, vocab=(ad, bd, vm))
    _note(compare(mx, g, label="xvocab duplicate map entries"))


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_xvocab_drafter_vocabulary_longer(gpu, dtype):
    """A drafter vocabulary much longer than the verifier's: rows take as
    many chunks as the drafter rows need."""
    from parity_util import make_xvocab
    x = synth.generate(B=4, K=3, V=3000, dtype=dtype, rho=("uniform", 0.0, 2.0),
                       tau=("alternate", 1.0, 0.7), seed=18)
    ad, bd, vm, mx = make_xvocab(x, 40000, 0.9, seed=3)
    g = run_gpu(mx, vocab=(ad, bd, vm), want_full=True, fuse_bonus=True)
    _note(compare(mx, g, fuse_bonus=True, label=f"xvocab Vd=40000 {dtype}"))
    compare_full(mx, g[4], fuse_bonus=True, label="xvocab Vd=40000 full")


# ------------------------------------------------------ the error path --
@pytest.mark.parametrize("B", [256, 257])
def test_polling_modes_at_the_boundary(gpu, B):
    """A launch of at most 4096 statistics items (4 per CU slot of the
    256-CU part) polls every slot it waits for, a larger one a sentinel slot
    first; B = 256 and 257 requests of 4 rows x 4 chunks sit on either side
    of that boundary, and both agree with the oracle."""
    x = synth.generate(B=B, K=3, V=60000, dtype="bf16", rho=("uniform", 0.0, 2.0),
                       tau=("alternate", 0.0, 1.0), seed=5150 + B)
    g = run_gpu(x)
    r = compare(x, g, label=f"polling boundary B={B}")
    _note(r)
    assert len(r["near_ties"]) <= near_tie_budget(x.B * (x.K + 1))


@pytest.mark.parametrize("B,K,V", [(24, 3, 20000), (288, 3, 60000)])
def test_timed_out_waits_mark_requests_invalid(gpu, B, K, V):
    """A wait bound of a few 10 ns ticks (set from the host) makes waits
    between workgroups run out under normal operation: the workspace counts
    them, and every request either carries accept_len = -1 or the oracle's
    outputs; with the default bound restored the same call is whole.  The
    small launch polls every slot it waits for, the large one (4608
    statistics items) a sentinel slot first."""
    import paper_2608_26004_amd as asp
    import torch
    from parity_util import to_device
    x = synth.generate(B=B, K=K, V=V, dtype="bf16", rho=("uniform", 0.0, 2.0),
                       tau=("alternate", 0.0, 1.0), seed=4242)
    args = [to_device(v) for v in (x.t, x.a, x.b, x.draft_tokens, x.draft_probs, x.uniforms,
                                   x.temperature)]
    ws = asp.Workspace(torch.device("cuda"))
    try:
        asp.set_wait_limit(2)
        acc, nxt, flp, gate = asp.fuse_verify(*args, return_gate=True, workspace=ws)
        torch.cuda.synchronize()
    finally:
        asp.set_wait_limit(0)
    n_to = ws.timeouts()
    acc, nxt, flp = acc.cpu().numpy(), nxt.cpu().numpy(), flp.cpu().numpy()
    acc_o, nxt_o, flp_o, _, res = O.fuse_verify(x.t, x.a, x.b, x.draft_tokens, x.draft_probs,
                                                x.uniforms, x.temperature)
    bad = acc == -1
    print(f"[timeouts] {n_to} timed-out waits, {int(bad.sum())} of {x.B} requests marked invalid")
    assert n_to > 0 and bad.any()
    for bi in np.nonzero(~bad)[0]:
        if res[bi].near_tie(1e-6):
            continue
        assert (acc[bi], nxt[bi]) == (acc_o[bi], nxt_o[bi]), bi
        assert np.abs(flp[bi] - flp_o[bi]).max() < 1e-5
    # default bound: no timeouts, full parity, on the same workspace
    before = ws.timeouts()
    g = asp.fuse_verify(*args, return_gate=True, workspace=ws)
    torch.cuda.synchronize()
    assert ws.timeouts() == before
    _note(compare(x, [v.cpu().numpy() for v in g], label="after the error path"))
