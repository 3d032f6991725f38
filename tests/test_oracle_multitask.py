"""Pins of the oracle's task-aware embedding (task, charge, spin and element
composition): central differences of the loss against every weight gradient;
zero tables reduce to the model without it; a single-element structure equals
the base model with a shifted species row; a label change moves only its own
structure's energy; the four table gradients share one total; permutation
invariance."""
import dataclasses

import numpy as np
import pytest

from oracle.model import (Params, build_graph, forces, forward_energy, loss_and_seeds, route_all,
                          training_step)
from oracle.neighbors import neighbor_list
from paper_2604_15821_amd.synth import _draw_weights, make_batch, subset

TABLES = ("Tk", "Qe", "Se", "Wc")


def _task_batch(n_struct=3, seed=12):
    b = make_batch("tiny", n_struct=n_struct)
    m = dataclasses.replace(b.model, n_tasks=3, n_charges=5, n_spins=2)
    rng = np.random.default_rng(seed)
    W = _draw_weights(rng, m, 0.0)
    S = b.n_struct
    return dataclasses.replace(b, model=m, weights=W, task=rng.integers(0, 3, S).astype(np.int32),
                               charge=rng.integers(0, 5, S).astype(np.int32),
                               spin=rng.integers(0, 2, S).astype(np.int32))


def _loss(b, weights, edges):
    m = b.model
    P = Params.from_weights(weights, m)
    g = build_graph(b.pos, b.cell, b.offsets, m.r_cut, m.n_rbf, edges, labels=(b.task, b.charge, b.spin))
    rt = route_all(b.species, g, P)
    E, cache = forward_energy(b.species, g, P, rt)
    F = forces(b.species, g, P, rt, cache)
    return loss_and_seeds(E, F, b.E_ref, b.F_ref, g.n_atoms_struct, m.w_E, m.w_F)[0]


def test_weight_gradient_matches_central_differences():
    b = _task_batch()
    edges = neighbor_list(b.pos, b.cell, b.offsets, b.model.r_cut)
    loss, E, F, grad = training_step(b, edges=edges)
    assert loss == pytest.approx(_loss(b, b.weights, edges), rel=1e-13)
    w64 = {k: v.astype(np.float64) for k, v in b.weights.items()}
    rng = np.random.default_rng(1)
    for name in TABLES + ("A", "W_o1", "blocks.0.W1", "blocks.1.W_b"):
        W = w64[name]
        picks = [tuple(int(i) for i in np.unravel_index(np.argmax(np.abs(grad[name])), W.shape))]
        picks += [tuple(int(rng.integers(0, s)) for s in W.shape) for _ in range(2)]
        for idx in picks:
            h = 1e-6 * max(1.0, abs(W[idx]))
            wp = dict(w64); wp[name] = W.copy(); wp[name][idx] += h
            wm = dict(w64); wm[name] = W.copy(); wm[name][idx] -= h
            fd = (_loss(b, wp, edges) - _loss(b, wm, edges)) / (2 * h)
            scale = max(np.abs(grad[name]).max(), 1e-12)
            assert abs(fd - grad[name][idx]) <= 2e-6 * scale + 1e-9, (name, idx, fd, grad[name][idx])
    for name in TABLES:
        assert np.abs(grad[name]).max() > 0


def test_zero_tables_reduce_to_the_base_model():
    b = _task_batch()
    W = dict(b.weights)
    for n in TABLES:
        W[n] = np.zeros_like(W[n])
    l1, E1, F1, g1 = training_step(dataclasses.replace(b, weights=W))
    m0 = dataclasses.replace(b.model, n_tasks=0, n_charges=0, n_spins=0)
    W0 = {k: v for k, v in W.items() if k not in TABLES}
    l0, E0, F0, g0 = training_step(dataclasses.replace(b, model=m0, weights=W0))
    np.testing.assert_allclose(E1, E0, rtol=1e-14)
    np.testing.assert_allclose(F1, F0, rtol=1e-12, atol=1e-14)
    for k, v in g0.items():
        np.testing.assert_allclose(g1[k], v, rtol=1e-12, atol=1e-14 * max(1.0, np.abs(v).max()), err_msg=k)


def test_single_element_structure_equals_a_shifted_species_row():
    """All atoms of element z: h0 = A[z] + Tk[t] + Qe[q] + Se[p] + Wc[z] for every atom,
    which the base model reproduces with that sum as its row z."""
    b = _task_batch(n_struct=1)
    z = 17
    b = dataclasses.replace(b, species=np.full(b.n_atoms, z, np.int32))
    W = b.weights
    t, q, p = int(b.task[0]), int(b.charge[0]), int(b.spin[0])
    A = W["A"].astype(np.float64).copy()
    W64 = {k: v.astype(np.float64) for k, v in W.items()}
    A[z] = A[z] + (((W64["Tk"][t] + W64["Qe"][q]) + W64["Se"][p]) + W64["Wc"][z])
    m0 = dataclasses.replace(b.model, n_tasks=0, n_charges=0, n_spins=0)
    W0 = {k: v for k, v in W.items() if k not in TABLES}
    W0["A"] = A
    l1, E1, F1, g1 = training_step(b)
    l0, E0, F0, g0 = training_step(dataclasses.replace(b, model=m0, weights=W0))
    np.testing.assert_allclose(E1, E0, rtol=1e-12)
    np.testing.assert_allclose(F1, F0, rtol=1e-9, atol=1e-12)


def test_a_label_moves_only_its_own_structure():
    b = _task_batch(n_struct=3)
    E0 = training_step(b)[1]
    task = b.task.copy()
    task[1] = (task[1] + 1) % 3
    E1 = training_step(dataclasses.replace(b, task=task))[1]
    assert E1[0] == E0[0] and E1[2] == E0[2]
    assert abs(E1[1] - E0[1]) > 1e-6


def test_table_gradients_share_one_total():
    """Each table row sum over its labels is the sum over structures of the adjoint of the
    per-structure vector (the composition fractions of a structure sum to one)."""
    b = _task_batch(n_struct=4)
    grad = training_step(b)[3]
    tot = grad["Tk"].sum(0)
    for n in ("Qe", "Se", "Wc"):
        np.testing.assert_allclose(grad[n].sum(0), tot, rtol=1e-10, atol=1e-12 * np.abs(tot).max())


def test_permutation_invariance():
    b = _task_batch(n_struct=2)
    l0, E0, F0, g0 = training_step(b)
    rng = np.random.default_rng(6)
    perm = np.concatenate([b.offsets[s] + rng.permutation(b.offsets[s + 1] - b.offsets[s])
                           for s in range(b.n_struct)])
    l1, E1, F1, g1 = training_step(dataclasses.replace(b, pos=b.pos[perm], species=b.species[perm],
                                                       F_ref=b.F_ref[perm]))
    np.testing.assert_allclose(E1, E0, rtol=1e-12)
    np.testing.assert_allclose(F1, F0[perm], rtol=1e-9, atol=1e-12)
    for k in g0:
        np.testing.assert_allclose(g1[k], g0[k], rtol=1e-9, atol=1e-12 * max(1.0, np.abs(g0[k]).max()))


def test_subset_keeps_the_labels():
    b = make_batch("multitask", n_struct=6)
    s = subset(b, [4, 1])
    assert (s.task == b.task[[4, 1]]).all() and (s.spin == b.spin[[4, 1]]).all()
