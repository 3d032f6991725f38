"""Pins of the oracle's feature-update (atom) MoE: finite differences of the
energy against the forces and of the loss against every weight gradient
(W1f, W2f, Pf included), the reduction to the model without it when its
experts output zero, a router that cannot receive gradient, routing by
element type against a brute-force sort, and permutation invariance."""
import dataclasses

import numpy as np
import pytest

from oracle.model import (Params, build_graph, forces, forward_energy, loss_and_seeds, route_all,
                          route_atoms, training_step)
from oracle.neighbors import neighbor_list
from paper_2604_15821_amd.synth import _draw_weights, make_batch

FIXED = ("beta", "beta3", "betaf")


def _fixed(name):
    return name.rsplit(".", 1)[-1] in FIXED


def _atom_batch(n_struct=2, name="tiny", seed=11, **changes):
    b = make_batch(name, n_struct=n_struct)
    kw = dict(atom_moe=True, n_experts_f=3, top_k_f=2, d_hidden_f=48)
    kw.update(changes)
    m = dataclasses.replace(b.model, **kw)
    return dataclasses.replace(b, model=m, weights=_draw_weights(np.random.default_rng(seed), m, 0.0))


def _energy(b, pos, edges, routing=None, weights=None):
    m = b.model
    P = Params.from_weights(b.weights if weights is None else weights, m)
    g = build_graph(pos, b.cell, b.offsets, m.r_cut, m.n_rbf, edges)
    rt = routing if routing is not None else route_all(b.species, g, P)
    E, cache = forward_energy(b.species, g, P, rt)
    return E, g, P, rt, cache


def test_forces_match_central_differences_of_energy():
    b = _atom_batch(3)
    pos = b.pos.astype(np.float64)
    edges = neighbor_list(b.pos, b.cell, b.offsets, b.model.r_cut)
    E, g, P, rt, cache = _energy(b, pos, edges)
    F = forces(b.species, g, P, rt, cache)
    rng = np.random.default_rng(0)
    h = 1e-5
    for a in rng.choice(pos.shape[0], 12, replace=False):
        for c in range(3):
            p1 = pos.copy(); p1[a, c] += h
            p2 = pos.copy(); p2[a, c] -= h
            fd = -(_energy(b, p1, edges, rt)[0].sum() - _energy(b, p2, edges, rt)[0].sum()) / (2 * h)
            assert abs(fd - F[a, c]) <= 1e-6 * max(1.0, abs(F[a, c]))


def _loss(b, weights, edges, routing_ref):
    m = b.model
    E, g, P, rt, cache = _energy(b, b.pos, edges, weights=weights)
    for r0, r1 in zip(routing_ref, rt):
        if not (np.array_equal(r0.eid, r1.eid) and np.array_equal(r0.atom.eid, r1.atom.eid)):
            return None
    F = forces(b.species, g, P, rt, cache)
    return loss_and_seeds(E, F, b.E_ref, b.F_ref, g.n_atoms_struct, m.w_E, m.w_F)[0]


@pytest.mark.parametrize("changes", [{}, {"n_experts_f": 4, "top_k_f": 1, "top_k": 1}],
                         ids=["Ef3-k2", "Ef4-k1"])
def test_weight_gradient_matches_central_differences(changes):
    b = _atom_batch(2, **changes)
    edges = neighbor_list(b.pos, b.cell, b.offsets, b.model.r_cut)
    loss, E, F, grad, aux = training_step(b, edges=edges, return_aux=True)
    w64 = {k: v.astype(np.float64) for k, v in b.weights.items()}
    rng = np.random.default_rng(2)
    checked = set()
    for name, W in w64.items():
        if _fixed(name):
            assert np.all(grad[name] == 0.0)
            continue
        picks = [tuple(int(i) for i in np.unravel_index(np.argmax(np.abs(grad[name])), W.shape))]
        picks += [tuple(int(rng.integers(0, s)) for s in W.shape) for _ in range(2)]
        for idx in picks:
            h = 1e-6 * max(1.0, abs(W[idx]))
            wp = dict(w64); wp[name] = W.copy(); wp[name][idx] += h
            wm = dict(w64); wm[name] = W.copy(); wm[name][idx] -= h
            lp, lm = _loss(b, wp, edges, aux["routing"]), _loss(b, wm, edges, aux["routing"])
            if lp is None or lm is None:
                continue                                       # +-h flips a top-k decision
            fd = (lp - lm) / (2 * h)
            scale = max(np.abs(grad[name]).max(), 1e-12)
            assert abs(fd - grad[name][idx]) <= 2e-6 * scale + 1e-9, (name, idx, fd, grad[name][idx])
            checked.add(name)
    for t in range(b.model.n_blocks):
        for n in ("W1f", "W2f", "Pf"):
            assert f"blocks.{t}.{n}" in checked


def test_zero_output_experts_reduce_to_the_model_without_the_atom_moe():
    """W2f = 0 makes every feature-update output zero: energies and forces equal those of
    the same model without the layer, and only W2f receives gradient inside it."""
    b = _atom_batch(2)
    w = dict(b.weights)
    for t in range(b.model.n_blocks):
        w[f"blocks.{t}.W2f"] = np.zeros_like(w[f"blocks.{t}.W2f"])
    b0 = dataclasses.replace(b, weights=w)
    loss0, E0, F0, g0 = training_step(b0)
    base_m = dataclasses.replace(b.model, atom_moe=False, n_experts_f=0, top_k_f=0, d_hidden_f=0)
    base_w = {k: v for k, v in w.items() if k.rsplit(".", 1)[-1] not in ("Pf", "betaf", "W1f", "W2f")}
    loss1, E1, F1, g1 = training_step(dataclasses.replace(b, model=base_m, weights=base_w))
    np.testing.assert_allclose(E0, E1, rtol=1e-14)
    np.testing.assert_allclose(F0, F1, rtol=1e-12, atol=1e-14)
    assert loss0 == pytest.approx(loss1, rel=1e-14)
    for k, v in g1.items():
        np.testing.assert_allclose(g0[k], v, rtol=1e-12, atol=1e-14 * max(1.0, np.abs(v).max()), err_msg=k)
    for t in range(b.model.n_blocks):
        assert np.all(g0[f"blocks.{t}.W1f"] == 0.0) and np.all(g0[f"blocks.{t}.Pf"] == 0.0)
        assert np.abs(g0[f"blocks.{t}.W2f"]).max() > 0.0


def test_single_feature_expert_router_gets_no_gradient():
    b = _atom_batch(2, n_experts_f=1, top_k_f=1)
    loss, E, F, grad = training_step(b)
    for t in range(b.model.n_blocks):
        assert np.abs(grad[f"blocks.{t}.Pf"]).max() < 1e-14
        assert np.abs(grad[f"blocks.{t}.W1f"]).max() > 0


def test_atom_routing_is_by_element_type_against_a_full_stable_sort():
    b = make_batch("atom_moe", n_struct=2)
    m = b.model
    w = b.weights
    for t in range(m.n_blocks):
        Pf, bf = w[f"blocks.{t}.Pf"], w[f"blocks.{t}.betaf"]
        rt = route_atoms(b.species, Pf, bf, m.top_k_f)
        l32 = Pf[b.species] + bf
        for i in range(b.n_atoms):
            want = sorted(range(m.n_experts_f), key=lambda x: (-float(l32[i, x]), x))[:m.top_k_f]
            assert rt.eid[i].tolist() == want
        for z in np.unique(b.species):                  # one expert set per element
            rows = rt.eid[b.species == z]
            assert (rows == rows[0]).all()
        assert rt.counts.sum() == b.n_atoms * m.top_k_f
        flat = rt.eid.reshape(-1)
        assert np.array_equal(rt.pos.reshape(-1)[rt.inv], np.arange(flat.size))
        assert np.all(np.diff(flat[rt.inv]) >= 0)
        np.testing.assert_allclose(rt.prob.sum(1), 1.0, rtol=1e-14)


def test_energy_invariant_under_atom_permutation():
    b = _atom_batch(3)
    loss0, E0, F0, g0 = training_step(b)
    rng = np.random.default_rng(6)
    perm = np.concatenate([b.offsets[s] + rng.permutation(b.offsets[s + 1] - b.offsets[s])
                           for s in range(b.n_struct)])
    b2 = dataclasses.replace(b, pos=b.pos[perm], species=b.species[perm], F_ref=b.F_ref[perm])
    loss1, E1, F1, g1 = training_step(b2)
    np.testing.assert_allclose(E1, E0, rtol=1e-12)
    np.testing.assert_allclose(F1, F0[perm], rtol=1e-9, atol=1e-12)
    for k in g0:
        np.testing.assert_allclose(g1[k], g0[k], rtol=1e-9, atol=1e-12 * max(1.0, np.abs(g0[k]).max()))
