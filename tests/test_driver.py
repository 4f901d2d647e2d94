"""Multi-step driver (Alg. 1's loop around the decision step): host logic
against closed forms, and the HIP step against the oracle over whole
trajectories."""

import numpy as np
import pytest

import oracle as O
from paper_2608_26004_amd import driver as drv
from paper_2608_26004_amd import synth


def oracle_step(beta=1.0, gamma=0.5, near=None):
    def fn(t, a, b, d, q, u, tau):
        acc, nxt, _, _, res = O.fuse_verify(t, a, b, d, q, u, tau, beta=beta, gamma=gamma)
        if near is not None:
            near.append([r.near_tie(1e-6) for r in res])
        return acc, nxt
    return fn


def greedy_decode(models, h0, n):
    """The verifier's own greedy decode from context hash h0."""
    out, h = [], h0
    for _ in range(n):
        tok = int(np.argmax(synth.stored_to_f64(models.host[0][int(models.row_index(h))])))
        out.append(tok)
        h = drv.roll(h, tok)
    return out


@pytest.mark.parametrize("dtype", [synth.BF16, synth.FP32])
def test_identical_views_greedy_is_verifier_greedy_decode(dtype):
    """With a = b = t (delta = 0, D = 0) the drafts are the verifier's argmax
    and Eq. 4 reads p_t(d) > gamma p_t(d): every draft is accepted (AR = 1,
    MAL = K + 1) and the committed text is the verifier's greedy decode."""
    K, B = 3, 3
    m = drv.TableModels(300, R=64, identical=True, dtype=dtype, seed=1)
    dec = drv.SpecDecoder(m, B, K, 0.0, backend="host", step_fn=oracle_step(), seed=2)
    h0 = dec.h.copy()
    for _ in range(5):
        dec.step()
    rep = dec.report()
    assert rep["AR"] == 1.0 and rep["MAL"] == K + 1
    for r in range(B):
        assert dec.tokens[r] == greedy_decode(m, h0[r], len(dec.tokens[r]))


def test_identical_views_sampling_accepts_everything():
    """Sampling form with a = t and the drafter's own q: the ratio is
    1 / gamma_eff >= 1, so every draft passes (AR = 1, MAL = K + 1)."""
    K, B = 4, 2
    m = drv.TableModels(200, R=32, identical=True, dtype=synth.FP32, seed=3)
    dec = drv.SpecDecoder(m, B, K, 1.0, backend="host", step_fn=oracle_step(), seed=4)
    for _ in range(4):
        dec.step()
    rep = dec.report()
    assert rep["AR"] == 1.0 and rep["MAL"] == K + 1


def test_report_definitions():
    """AR counts the drafts Alg. 1 evaluates (accepted ones plus the first
    rejection); MAL the tokens committed per step (accept_len + 1)."""
    K = 3
    script = iter([np.array([0, 3, 1]), np.array([2, 0, 3])])
    m = drv.TableModels(50, R=8, dtype=synth.FP32, seed=5)

    def fn(t, a, b, d, q, u, tau):
        return next(script), np.zeros(3, np.int32)

    dec = drv.SpecDecoder(m, 3, K, 0.0, backend="host", step_fn=fn, seed=6)
    dec.step()
    dec.step()
    acc = [0, 3, 1, 2, 0, 3]
    ev = sum(j + (1 if j < K else 0) for j in acc)
    rep = dec.report()
    assert rep["AR"] == sum(acc) / ev
    assert rep["MAL"] == sum(j + 1 for j in acc) / 6
    assert rep["tokens"] == sum(j + 1 for j in acc)


def test_trajectories_are_deterministic():
    m = drv.TableModels(400, R=64, rho=1.0, seed=7)
    runs = []
    for _ in range(2):
        dec = drv.SpecDecoder(m, 3, 2, np.array([0.0, 1.0, 0.7]), backend="host",
                              step_fn=oracle_step(), seed=8)
        for _ in range(4):
            dec.step()
        runs.append([list(x) for x in dec.tokens])
    assert runs[0] == runs[1]


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", [synth.BF16, synth.FP32])
def test_hip_trajectory_matches_oracle(dtype):
    """The same loop with the HIP step and with the oracle step, in
    lockstep: identical accept lengths and tokens at every step (a request
    whose oracle decision is a near tie may legitimately diverge; it is
    dropped from the comparison from then on)."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    dev = torch.device("cuda")
    m = drv.TableModels(3000, R=128, rho=1.5, dtype=dtype, seed=11, device=dev)
    tau = np.array([0.0, 1.0, 0.7, 0.0, 1.0, 0.0])
    g = drv.SpecDecoder(m, 6, 3, tau, seed=12, device=dev)
    near = []
    c = drv.SpecDecoder(m, 6, 3, tau, seed=12, backend="host", step_fn=oracle_step(near=near))
    live = np.ones(6, bool)
    for s in range(15):
        ag, ng = g.step()
        ac, nc = c.step()
        same = (ag == ac) & (ng == nc)
        bad = live & ~same & ~np.array(near[-1])
        assert not bad.any(), f"step {s}: hip {ag.tolist()} {ng.tolist()} oracle {ac.tolist()} {nc.tolist()}"
        live &= same
    assert live.sum() >= 5
    for r in np.nonzero(live)[0]:
        assert g.tokens[r] == c.tokens[r]
    print(f"[driver] {dtype}: hip {g.report()} oracle {c.report()}")
