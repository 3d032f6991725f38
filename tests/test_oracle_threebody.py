"""Pins of the oracle's three-body (bond-angle) term: feature derivatives
against finite differences, forces against central differences of the
energy, weight gradients against central differences of the loss, the
directional derivative, invariances, zero net force and smoothness where a
bond crosses the three-body cutoff."""
import dataclasses

import numpy as np
import pytest

from oracle import threebody as tb
from oracle.basis import bessel_basis, legendre
from oracle.model import (Params, build_graph, energy_tangent, forces, forward_energy, loss_and_seeds,
                          route_all, training_step)
from oracle.neighbors import neighbor_list
from paper_2604_15821_amd.synth import _draw_weights, make_batch, subset


def _batch(n_struct=1, **changes):
    b = subset(make_batch("threebody"), range(n_struct))
    m = dataclasses.replace(b.model, d=64, d_hidden=128, n_experts=4, top_k=2, n_experts3=4, top_k3=2,
                            d_hidden3=64, n_rbf=8, n_blocks=2, **changes)
    return dataclasses.replace(b, model=m, weights=_draw_weights(np.random.default_rng(7), m, 0.0))


def _three(m):
    return (m.r_cut3, m.n_legendre)


def _energy(b, pos, edges, routing=None, weights=None):
    m = b.model
    P = Params.from_weights(weights or b.weights, m)
    g = build_graph(pos, b.cell, b.offsets, m.r_cut, m.n_rbf, edges, _three(m))
    rt = routing if routing is not None else route_all(b.species, g, P)
    E, cache = forward_energy(b.species, g, P, rt)
    return E, g, P, rt, cache


def test_feature_partials_match_finite_differences():
    rng = np.random.default_rng(0)
    r3, nb, nl = 3.5, 6, 5
    # two edges out of one centre: e = 0, e2 = 1
    d = np.array([[1.1, 0.7, -0.4], [-0.3, 1.9, 0.8]])
    def feats(d):
        r = np.sqrt((d * d).sum(1))
        u = d / r[:, None]
        return tb.triplet_features(np.array([0]), np.array([1]), np.array([0, 1, 1]), r, u, r3, nb, nl), r, u
    tri, r, u = feats(d)
    # tangent along a random displacement vs central differences
    dd = rng.standard_normal(d.shape)
    h = 1e-6
    fd = (feats(d + h * dd)[0].G - feats(d - h * dd)[0].G) / (2 * h)
    an = tb.feature_tangent(tri, r, u, dd)
    assert np.abs(fd - an).max() <= 1e-7 * max(1.0, np.abs(an).max())
    # the displacement adjoint is the transpose of the tangent
    Gbar = rng.standard_normal(tri.G.shape)
    adj = tb.displacement_adjoint(tri, r, u, Gbar, 2)
    assert abs((adj * dd).sum() - (Gbar * an).sum()) <= 1e-10 * abs((Gbar * an).sum())


def test_features_closed_forms():
    r3, nb, nl = 3.5, 4, 5
    # collinear bonds: P_l(1) = 1, so every Legendre row equals B3(r2) u(r1 / r3)
    d = np.array([[1.0, 0.0, 0.0], [2.0, 0.0, 0.0]])
    r = np.sqrt((d * d).sum(1)); u = d / r[:, None]
    tri = tb.triplet_features(np.array([0]), np.array([1]), np.array([0, 1, 1]), r, u, r3, nb, nl)
    B3 = bessel_basis(r[1:], r3, nb)[0][0]
    x = r[0] / r3
    env = 1 - 28 * x ** 6 + 48 * x ** 7 - 21 * x ** 8
    np.testing.assert_allclose(tri.G.reshape(nl, nb), np.tile(B3 * env, (nl, 1)), rtol=1e-14)
    # orthogonal bonds: c = 0 and P_1(0) = P_3(0) = 0
    d = np.array([[1.0, 0.0, 0.0], [0.0, 2.0, 0.0]])
    r = np.sqrt((d * d).sum(1)); u = d / r[:, None]
    tri = tb.triplet_features(np.array([0]), np.array([1]), np.array([0, 1, 1]), r, u, r3, nb, nl)
    G = tri.G.reshape(nl, nb)
    assert tri.c[0] == 0.0 and np.abs(G[1]).max() == 0.0 and np.abs(G[3]).max() == 0.0
    P, _ = legendre(np.array([0.0]), nl)
    np.testing.assert_allclose(G[2], P[0, 2] * G[0], rtol=1e-14)


def test_forces_match_central_differences_with_angles():
    b = _batch(1)
    pos = b.pos.astype(np.float64)
    edges = neighbor_list(b.pos, b.cell, b.offsets, b.model.r_cut)
    E, g, P, rt, cache = _energy(b, pos, edges)
    assert g.tri.te.size > 100
    F = forces(b.species, g, P, rt, cache)
    rng = np.random.default_rng(0)
    h = 1e-5
    for a in rng.choice(pos.shape[0], 8, replace=False):
        for c in range(3):
            p1 = pos.copy(); p1[a, c] += h
            p2 = pos.copy(); p2[a, c] -= h
            fd = -(_energy(b, p1, edges, rt)[0].sum() - _energy(b, p2, edges, rt)[0].sum()) / (2 * h)
            assert abs(fd - F[a, c]) <= 1e-6 * max(1.0, abs(F[a, c])), (a, c, fd, F[a, c])


def test_three_body_part_is_not_negligible():
    b = _batch(1)
    loss, E, F, grad = training_step(b)
    b0 = dataclasses.replace(b, weights={**b.weights, **{k: np.zeros_like(v) for k, v in b.weights.items()
                                                         if k.endswith("W2a")}})
    _, E0, F0, _ = training_step(b0)
    assert np.linalg.norm(F - F0) > 0.05 * np.linalg.norm(F)


def test_net_force_zero_and_directional_derivative():
    b = _batch(2)
    pos = b.pos.astype(np.float64)
    edges = neighbor_list(b.pos, b.cell, b.offsets, b.model.r_cut)
    E, g, P, rt, cache = _energy(b, pos, edges)
    F = forces(b.species, g, P, rt, cache)
    for s in range(b.n_struct):
        Fs = F[b.offsets[s]:b.offsets[s + 1]]
        assert np.abs(Fs.sum(0)).max() <= 1e-12 * np.abs(Fs).max() * Fs.shape[0]
    phi = np.random.default_rng(1).standard_normal(pos.shape)
    dphi, _ = energy_tangent(b.species, g, P, rt, phi)
    assert abs(dphi + (phi * F).sum()) <= 1e-10 * abs(dphi)
    eps = 1e-6
    fd = (_energy(b, pos + eps * phi, edges, rt)[0].sum() - _energy(b, pos - eps * phi, edges, rt)[0].sum()) / (2 * eps)
    assert abs(fd - dphi) <= 1e-6 * abs(dphi)


def test_weight_gradient_matches_central_differences_with_angles():
    b = _batch(1)
    m = b.model
    edges = neighbor_list(b.pos, b.cell, b.offsets, m.r_cut)
    loss, E, F, grad, aux = training_step(b, edges=edges, return_aux=True)
    w64 = {k: v.astype(np.float64) for k, v in b.weights.items()}

    def L(w):
        P = Params.from_weights(w, m)
        g = build_graph(b.pos, b.cell, b.offsets, m.r_cut, m.n_rbf, edges, _three(m))
        rt = route_all(b.species, g, P)
        for r0, r1 in zip(aux["routing"], rt):
            if not (np.array_equal(r0.eid, r1.eid) and np.array_equal(r0.tri.eid, r1.tri.eid)):
                return None
        E_, c_ = forward_energy(b.species, g, P, rt)
        F_ = forces(b.species, g, P, rt, c_)
        return loss_and_seeds(E_, F_, b.E_ref, b.F_ref, g.n_atoms_struct, m.w_E, m.w_F)[0]

    rng = np.random.default_rng(3)
    checked = 0
    for name, W in w64.items():
        if name.endswith("beta") or name.endswith("beta3"):
            assert np.all(grad[name] == 0.0)
            continue
        picks = [tuple(int(i) for i in np.unravel_index(np.argmax(np.abs(grad[name])), W.shape))]
        picks += [tuple(int(rng.integers(0, s)) for s in W.shape)]
        for idx in picks:
            h = 1e-6 * max(1.0, abs(W[idx]))
            wp = dict(w64); wp[name] = W.copy(); wp[name][idx] += h
            wm = dict(w64); wm[name] = W.copy(); wm[name][idx] -= h
            lp, lm = L(wp), L(wm)
            if lp is None or lm is None:
                continue
            fd = (lp - lm) / (2 * h)
            scale = max(np.abs(grad[name]).max(), 1e-12)
            assert abs(fd - grad[name][idx]) <= 2e-6 * scale + 1e-9, (name, idx, fd, grad[name][idx])
            checked += 1
    assert checked >= 2 * len(w64) - 10


def _rotation(rng):
    q, r = np.linalg.qr(rng.standard_normal((3, 3)))
    q = q * np.sign(np.diag(r))
    return q if np.linalg.det(q) > 0 else -q


def test_energy_invariant_under_rotation_translation_permutation():
    b = _batch(1)
    m = b.model
    E0 = training_step(b)[1]
    rng = np.random.default_rng(5)
    # rotation of a periodic structure: rotate positions and cell together (triclinic cell)
    R = _rotation(rng)
    P = Params.from_weights(b.weights, m)
    pos_r = b.pos.astype(np.float64) @ R.T
    cell_r = b.cell.astype(np.float64) @ R.T
    # the neighbour list is taken from the unrotated structure (same edges, rotated geometry)
    edges = neighbor_list(b.pos, b.cell, b.offsets, m.r_cut)
    g = build_graph(pos_r, cell_r, b.offsets, m.r_cut, m.n_rbf, edges, _three(m))
    E1, _ = forward_energy(b.species, g, P, route_all(b.species, g, P))
    assert abs(E1[0] - E0[0]) <= 1e-12 * max(1.0, abs(E0[0]))
    # translation
    g = build_graph(b.pos.astype(np.float64) + np.array([0.3, -1.7, 2.2]), b.cell, b.offsets, m.r_cut, m.n_rbf,
                    edges, _three(m))
    E2, _ = forward_energy(b.species, g, P, route_all(b.species, g, P))
    assert abs(E2[0] - E0[0]) <= 1e-12 * max(1.0, abs(E0[0]))
    # permutation of the atoms
    perm = rng.permutation(b.n_atoms)
    bp = dataclasses.replace(b, pos=b.pos[perm], species=b.species[perm], F_ref=b.F_ref[perm])
    E3 = training_step(bp)[1]
    assert abs(E3[0] - E0[0]) <= 1e-12 * max(1.0, abs(E0[0]))


def test_energy_is_smooth_where_a_bond_crosses_the_three_body_cutoff():
    # an isolated trimer: atom 1 on a bond of length sweeping across r3
    m = dataclasses.replace(_batch(1).model, r_cut=6.0)
    w = _draw_weights(np.random.default_rng(11), m, 0.0)
    r3 = m.r_cut3

    def energy(x):
        pos = np.array([[10.0, 10.0, 10.0], [10.0 + x, 10.0, 10.0], [10.0, 12.0, 10.4]], np.float32)
        bb = dataclasses.replace(_batch(1), model=m, weights=w, pos=pos, cell=np.diag([40.0] * 3)[None].astype(np.float32),
                                 species=np.array([3, 7, 11], np.int32), offsets=np.array([0, 3], np.int32),
                                 E_ref=np.zeros(1, np.float32), F_ref=np.zeros((3, 3), np.float32))
        return training_step(bb)[1][0]

    # second differences on a grid across r3: a jump (or a kink) at the cutoff
    # would give one of size ~J (or ~J' h) there, far above the smooth h^2 E''
    h = 1e-3
    E = np.array([energy(r3 + (k + 0.5) * h) for k in range(-6, 6)])
    d2 = np.abs(E[2:] - 2 * E[1:-1] + E[:-2])
    away = max(d2[0], d2[1], d2[-1], d2[-2])
    assert d2.max() <= 10 * away + 1e-13, d2
