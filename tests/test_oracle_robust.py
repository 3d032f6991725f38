"""Pins of the oracle's robust multi-task loss (paper Sec. "Multi-task training
strategies"): its seeds against central differences of the loss itself, its
reduction to the mean-squared loss, the Huber pieces and the weight's range, and
the whole step's weight gradient against central differences of the loss."""
import dataclasses
import math

import numpy as np
import pytest

from oracle.model import (huber2, loss_and_seeds, robust_loss_and_seeds, robust_weight, stress_loss_and_seed,
                          training_step)


def _inputs(rng, S=7, outlier=True):
    n = rng.integers(3, 9, S)
    offsets = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    N = int(offsets[-1])
    E = rng.normal(size=S) * n
    F = rng.normal(size=(N, 3))
    E_ref = rng.normal(size=S)
    F_ref = rng.normal(size=(N, 3))
    if outlier:
        E[2] += 12.0 * n[2]   # one structure far off: z beyond tau
    sigma = rng.normal(size=(S, 3, 3)) * 0.3
    S_ref = rng.normal(size=(S, 3, 3)) * 0.3
    return offsets, E, F, E_ref, F_ref, sigma, S_ref


@pytest.mark.parametrize("task", [None, "two"])
@pytest.mark.parametrize("w_S", [0.0, 0.7])
def test_seeds_match_central_differences(task, w_S):
    rng = np.random.default_rng(3)
    offsets, E, F, E_ref, F_ref, sigma, S_ref = _inputs(rng)
    S = E.size
    tk = None if task is None else (np.arange(S) % 2).astype(np.int32)
    kw = dict(task=tk, sigma=sigma, S_ref=S_ref, w_S=w_S)
    delta, tau = 0.8, 0.9

    def f(E_, F_, sig_):
        return robust_loss_and_seeds(E_, F_, E_ref, F_ref, offsets, 1.3, 0.7, delta, tau,
                                     **{**kw, "sigma": sig_})[0]

    loss, lam, phi, psi, aux = robust_loss_and_seeds(E, F, E_ref, F_ref, offsets, 1.3, 0.7, delta, tau, **kw)
    assert (aux["W"] < 0.999).any() and (aux["W"] == 1.0).any()   # both regimes are exercised
    h = 1e-6
    for s in range(S):
        ep, em = E.copy(), E.copy()
        ep[s] += h
        em[s] -= h
        fd = (f(ep, F, sigma) - f(em, F, sigma)) / (2 * h)
        assert abs(fd - lam[s]) <= 1e-6 * max(1.0, abs(lam[s])), (s, fd, lam[s])
    for a in range(0, F.shape[0], 3):
        for c in range(3):
            fp, fm = F.copy(), F.copy()
            fp[a, c] += h
            fm[a, c] -= h
            fd = (f(E, fp, sigma) - f(E, fm, sigma)) / (2 * h)
            assert abs(fd - phi[a, c]) <= 1e-6 * max(1.0, abs(phi[a, c])), (a, c, fd, phi[a, c])
    if w_S:
        for s in range(S):
            for q in (0, 4, 5):
                sp, sm = sigma.copy(), sigma.copy()
                sp.reshape(S, 9)[s, q] += h
                sm.reshape(S, 9)[s, q] -= h
                fd = (f(E, F, sp) - f(E, F, sm)) / (2 * h)
                assert abs(fd - psi.reshape(S, 9)[s, q]) <= 1e-6 * max(1.0, abs(psi.reshape(S, 9)[s, q]))


def test_reduces_to_mean_squared_loss():
    """No down-weighting (tau = inf), no Huber clip (delta = inf) and equal structure
    sizes: the robust loss is the mean-squared loss, seeds included."""
    rng = np.random.default_rng(5)
    S, n = 6, 5
    offsets = np.arange(0, (S + 1) * n, n, dtype=np.int32)
    E, E_ref = rng.normal(size=S) * n, rng.normal(size=S)
    F, F_ref = rng.normal(size=(S * n, 3)), rng.normal(size=(S * n, 3))
    sigma, S_ref = rng.normal(size=(S, 3, 3)), rng.normal(size=(S, 3, 3))
    loss, lam, phi, psi, aux = robust_loss_and_seeds(E, F, E_ref, F_ref, offsets, 1.1, 0.6, math.inf, math.inf,
                                                     sigma=sigma, S_ref=S_ref, w_S=0.4)
    l0, lam0, phi0 = loss_and_seeds(E, F, E_ref, F_ref, np.diff(offsets), 1.1, 0.6)
    lS, psi0 = stress_loss_and_seed(sigma, S_ref, S, 0.4)
    assert (aux["W"] == 1.0).all()
    assert abs(loss - (l0 + lS)) <= 1e-13 * abs(l0 + lS)
    np.testing.assert_allclose(lam, lam0, rtol=1e-13)
    np.testing.assert_allclose(phi, phi0, rtol=1e-13)
    np.testing.assert_allclose(psi, psi0, rtol=1e-13)


def test_huber_pieces():
    r = np.array([-3.0, -1.0, -0.25, 0.0, 0.5, 1.0, 2.5])
    rho, d = huber2(r, 1.0)
    np.testing.assert_array_equal(rho, [5.0, 1.0, 0.0625, 0.0, 0.25, 1.0, 4.0])
    np.testing.assert_array_equal(d, [-2.0, -2.0, -0.5, 0.0, 1.0, 2.0, 2.0])


def test_weight_is_one_in_the_normal_range_and_decays_beyond():
    z = np.array([-5.0, 0.0, 2.0, 2.5, 3.0, 6.0, 60.0])
    W, dW = robust_weight(z, 2.0)
    assert (W[:3] == 1.0).all() and (dW[:3] == 0.0).all()
    assert (np.diff(W[2:]) < 0).all() and W[-1] == 0.0
    np.testing.assert_allclose(W[3], math.exp(-0.125), rtol=1e-15)


def test_equal_losses_give_unit_weights():
    """All structures with the same base loss: sd = 0, z = 0, every weight 1."""
    S, n = 4, 3
    offsets = np.arange(0, (S + 1) * n, n, dtype=np.int32)
    E = np.full(S, 2.0 * n)
    F = np.ones((S * n, 3))
    loss, lam, phi, psi, aux = robust_loss_and_seeds(E, F, np.zeros(S), np.zeros((S * n, 3)), offsets, 1.0, 1.0,
                                                     math.inf, 2.0)
    assert (aux["z"] == 0.0).all() and (aux["W"] == 1.0).all()
    assert abs(loss - (4.0 + 1.0)) <= 1e-14


def test_weight_gradient_matches_central_differences():
    """The whole step with the robust loss: dL/dW of every weight tensor (its largest
    entry and two random ones) against central differences of the robust loss (tiny
    model, 4 structures, tau low enough that one structure is down-weighted)."""
    from oracle.model import Params, build_graph, forces, forward_energy, route_all
    from oracle.neighbors import neighbor_list
    from paper_2604_15821_amd.synth import make_batch, subset
    b = subset(make_batch("tiny"), range(4))
    m = dataclasses.replace(b.model, robust=1, huber_delta=0.5, robust_tau=0.6)
    b = dataclasses.replace(b, model=m)
    edges = neighbor_list(b.pos, b.cell, b.offsets, m.r_cut)
    loss, E, F, grad, aux = training_step(b, edges=edges, return_aux=True)
    W0 = robust_loss_and_seeds(E, F, b.E_ref, b.F_ref, b.offsets, m.w_E, m.w_F, m.huber_delta, m.robust_tau)[4]["W"]
    assert (W0 < 1.0).any()

    def lossat(weights):
        P = Params.from_weights(weights, m)
        g = build_graph(b.pos, b.cell, b.offsets, m.r_cut, m.n_rbf, edges)
        rt = route_all(b.species, g, P)
        for r0, r1 in zip(aux["routing"], rt):
            if not np.array_equal(r0.eid, r1.eid):
                return None
        E_, cache = forward_energy(b.species, g, P, rt)
        F_ = forces(b.species, g, P, rt, cache)
        return robust_loss_and_seeds(E_, F_, b.E_ref, b.F_ref, b.offsets, m.w_E, m.w_F, m.huber_delta,
                                     m.robust_tau)[0]

    w64 = {k: v.astype(np.float64) for k, v in b.weights.items()}
    assert abs(lossat(w64) - loss) <= 1e-12 * abs(loss)
    rng = np.random.default_rng(2)
    checked = 0
    for name_, W in w64.items():
        if name_.endswith("beta"):
            assert np.all(grad[name_] == 0.0)
            continue
        picks = [tuple(int(i) for i in np.unravel_index(np.argmax(np.abs(grad[name_])), W.shape))]
        picks += [tuple(int(rng.integers(0, s)) for s in W.shape) for _ in range(2)]
        for idx in picks:
            h = 1e-6 * max(1.0, abs(W[idx]))
            wp = dict(w64); wp[name_] = W.copy(); wp[name_][idx] += h
            wm = dict(w64); wm[name_] = W.copy(); wm[name_][idx] -= h
            lp, lm = lossat(wp), lossat(wm)
            if lp is None or lm is None:
                continue
            fd = (lp - lm) / (2 * h)
            scale = max(np.abs(grad[name_]).max(), 1e-12)
            assert abs(fd - grad[name_][idx]) <= 2e-6 * scale + 1e-9, (name_, idx, fd, grad[name_][idx])
            checked += 1
    assert checked >= 3 * len(w64) - 10
