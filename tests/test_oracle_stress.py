"""Pins of the oracle's stress and of the stress term of the loss:
sigma = (1/V) dE/deps against central differences of the energy under a
strain of positions and cell (with and without the bond-angle term),
symmetry, the dimer closed form, central differences of the loss with the
stress term against dL/dW, w_S = 0 leaving the step unchanged, and a torch
float64 implementation with stress and weight gradients from autograd."""
import dataclasses

import numpy as np
import pytest

from oracle.model import (Params, build_graph, build_graph_for, energy_displacement_gradient, forward_energy,
                          loss_and_seeds, route_all, stress, stress_loss_and_seed, training_step)
from oracle.neighbors import neighbor_list
from paper_2604_15821_amd.synth import Batch, _draw_weights, make_batch, subset

W_S = 0.1 * 160.2177 ** 2


def _strained_energy(b, eps, edges, routing, three=None):
    """Energies with every structure strained by (I + eps_s): positions and cell rows."""
    m = b.model
    A = np.eye(3)[None] + eps
    sid = np.repeat(np.arange(b.n_struct), np.diff(b.offsets))
    pos = np.einsum("nab,nb->na", A[sid], b.pos.astype(np.float64))
    cell = np.einsum("sab,scb->sca", A, b.cell.astype(np.float64))
    P = Params.from_weights(b.weights, m)
    g = build_graph(pos, cell, b.offsets, m.r_cut, m.n_rbf, edges, three)
    return forward_energy(b.species, g, P, routing)[0]


def _check_stress_by_differences(b, three=None, rtol=1e-6):
    m = b.model
    edges = neighbor_list(b.pos, b.cell, b.offsets, m.r_cut)
    loss, E, F, grad, aux = training_step(b, edges=edges, return_aux=True)
    sig = aux["stress"]
    V = np.abs(np.linalg.det(b.cell.astype(np.float64)))
    h = 1e-6
    for a in range(3):
        for c in range(3):
            e = np.zeros((b.n_struct, 3, 3))
            e[:, a, c] = h
            fd = (_strained_energy(b, e, edges, aux["routing"], three)
                  - _strained_energy(b, -e, edges, aux["routing"], three)) / (2 * h) / V
            np.testing.assert_allclose(sig[:, a, c], fd, rtol=rtol, atol=1e-9 * np.abs(sig).max())
    np.testing.assert_allclose(sig, sig.transpose(0, 2, 1), rtol=1e-10, atol=1e-14)   # rotation invariance
    assert np.abs(sig).max() > 1e-4
    return sig


def test_stress_matches_strain_differences():
    _check_stress_by_differences(make_batch("tiny", n_struct=3))


def test_stress_matches_strain_differences_with_angles():
    b = subset(make_batch("threebody"), range(1))
    m = dataclasses.replace(b.model, d=64, d_hidden=128, n_experts=4, n_experts3=4, d_hidden3=64, n_rbf=8,
                            n_blocks=2)
    b = dataclasses.replace(b, model=m, weights=_draw_weights(np.random.default_rng(7), m, 0.0))
    _check_stress_by_differences(b, three=(m.r_cut3, m.n_legendre), rtol=1e-5)


def test_dimer_stress_closed_form():
    """Two atoms in a large box: sigma = (1/V) (dE/dr) r rhat rhat^T."""
    m = make_batch("tiny").model
    W = _draw_weights(np.random.default_rng(8), m, 0.0)
    L = 30.0
    rhat = np.array([0.6, 0.0, 0.8])

    def dimer(r):
        pos = np.array([[10.0, 10.0, 10.0], 10.0 + r * rhat])
        b = Batch(pos=pos, cell=np.diag([L, L, L])[None].astype(np.float32),
                  species=np.array([7, 29], np.int32), offsets=np.array([0, 2], np.int32),
                  E_ref=np.zeros(1, np.float32), F_ref=np.zeros((2, 3), np.float32), weights=W, model=m,
                  S_ref=np.zeros((1, 3, 3), np.float32))
        return training_step(b, return_aux=True)
    r, h = 2.7, 1e-5
    sig = dimer(r)[4]["stress"][0]
    dEdr = (dimer(r + h)[1][0] - dimer(r - h)[1][0]) / (2 * h)
    np.testing.assert_allclose(sig, dEdr * r * np.outer(rhat, rhat) / L ** 3, rtol=1e-7, atol=1e-16)


def _loss(b, weights, edges, routing_ref):
    m = b.model
    P = Params.from_weights(weights, m)
    g = build_graph(b.pos, b.cell, b.offsets, m.r_cut, m.n_rbf, edges)
    rt = route_all(b.species, g, P)
    for r0, r1 in zip(routing_ref, rt):
        if not np.array_equal(r0.eid, r1.eid):
            return None
    E, cache = forward_energy(b.species, g, P, rt)
    G = energy_displacement_gradient(b.species, g, P, rt, cache)
    F = np.zeros((b.n_atoms, 3))
    np.add.at(F, g.ei, G)
    np.add.at(F, g.ej, -G)
    loss = loss_and_seeds(E, F, b.E_ref, b.F_ref, g.n_atoms_struct, m.w_E, m.w_F)[0]
    return loss + stress_loss_and_seed(stress(g, G, b.cell), b.S_ref, b.n_struct, m.w_S)[0]


def test_weight_gradient_with_stress_term_matches_central_differences():
    b = make_batch("tiny", n_struct=2)
    b = dataclasses.replace(b, model=dataclasses.replace(b.model, w_S=W_S))
    edges = neighbor_list(b.pos, b.cell, b.offsets, b.model.r_cut)
    loss, E, F, grad, aux = training_step(b, edges=edges, return_aux=True)
    assert loss == pytest.approx(_loss(b, b.weights, edges, aux["routing"]), rel=1e-13)
    w64 = {k: v.astype(np.float64) for k, v in b.weights.items()}
    rng = np.random.default_rng(3)
    checked = 0
    for name, W in w64.items():
        if name.endswith("beta"):
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
                continue
            fd = (lp - lm) / (2 * h)
            scale = max(np.abs(grad[name]).max(), 1e-12)
            assert abs(fd - grad[name][idx]) <= 2e-6 * scale + 1e-9, (name, idx, fd, grad[name][idx])
            checked += 1
    assert checked >= 3 * len(w64) - 12
    # the stress term changes the gradient well beyond the tolerances used against the GPU
    g0 = training_step(dataclasses.replace(b, model=dataclasses.replace(b.model, w_S=0.0)), edges=edges)[3]
    for name in ("W_o1", "blocks.0.W1", "blocks.1.W_b"):
        assert np.linalg.norm(grad[name] - g0[name]) > 1e-2 * np.linalg.norm(g0[name]), name


def test_zero_stress_weight_leaves_the_step_unchanged():
    b = make_batch("tiny", n_struct=2)
    l0, E0, F0, g0 = training_step(b)
    b1 = dataclasses.replace(b, S_ref=None)
    l1, E1, F1, g1 = training_step(b1)
    assert l0 == l1 and (E0 == E1).all() and (F0 == F1).all()
    for k in g0:
        assert (g0[k] == g1[k]).all()


torch = pytest.importorskip("torch")


def test_stress_and_loss_gradient_match_torch_autograd():
    """Energy written with torch ops on strained positions and cell; stress from
    autograd of the strain, forces from autograd of the positions, the loss with
    both and its weight gradient from a second autograd pass."""
    b = make_batch("tiny", n_struct=3)
    b = dataclasses.replace(b, model=dataclasses.replace(b.model, w_S=W_S))
    loss, E, F, grad, aux = training_step(b, return_aux=True)
    g, rts, m = aux["graph"], aux["routing"], b.model
    dt = torch.float64
    S = b.n_struct
    pos = torch.tensor(b.pos, dtype=dt, requires_grad=True)
    eps = torch.zeros(S, 3, 3, dtype=dt, requires_grad=True)
    W = {k: torch.tensor(v, dtype=dt, requires_grad=not k.endswith("beta")) for k, v in b.weights.items()}
    Z = torch.tensor(b.species, dtype=torch.long)
    ei, ej = torch.tensor(g.ei, dtype=torch.long), torch.tensor(g.ej, dtype=torch.long)
    sid = torch.tensor(g.struct_of_atom, dtype=torch.long)
    A = torch.eye(3, dtype=dt)[None] + eps
    ps = torch.einsum("nab,nb->na", A[sid], pos)
    cell = torch.einsum("sab,scb->sca", A, torch.tensor(b.cell, dtype=dt))
    d = ps[ej] - ps[ei] + torch.einsum("ek,ekc->ec", torch.tensor(g.shift, dtype=dt), cell[sid[ei]])
    r = torch.sqrt((d * d).sum(1))
    n = torch.arange(1, m.n_rbf + 1, dtype=dt)
    x = r / m.r_cut
    u = 1 - 28 * x ** 6 + 48 * x ** 7 - 21 * x ** 8
    B = (2.0 / m.r_cut) ** 0.5 * torch.sin(n[None] * np.pi * r[:, None] / m.r_cut) / r[:, None] * u[:, None]
    h = W["A"][Z]
    for t in range(m.n_blocks):
        p = f"blocks.{t}."
        X = (B @ W[p + "W_b"]) * h[ej]
        prob = torch.softmax(W[p + "Pc"][Z[ei]] + W[p + "Pn"][Z[ej]] + W[p + "beta"], dim=1)
        eid = torch.tensor(rts[t].eid, dtype=torch.long)
        msg = torch.zeros_like(X)
        for c in range(m.top_k):
            for xx in range(m.n_experts):
                rows = torch.nonzero(eid[:, c] == xx).flatten()
                if rows.numel():
                    y = torch.nn.functional.silu(X[rows] @ W[p + "W1"][xx]) @ W[p + "W2"][xx]
                    msg = msg.index_add(0, rows, prob[rows, xx][:, None] * y)
        h = h.index_add(0, ei, msg)
    eps_i = torch.nn.functional.silu(h @ W["W_o1"]) @ W["w_o2"]
    Es = torch.zeros(S, dtype=dt).index_add(0, sid, eps_i)
    dEdR, dEde = torch.autograd.grad(Es.sum(), [pos, eps], create_graph=True)
    V = torch.tensor(np.abs(np.linalg.det(b.cell.astype(np.float64))), dtype=dt)
    sig = dEde / V[:, None, None]
    Ft = -dEdR
    nat = torch.tensor(np.diff(b.offsets), dtype=dt)
    Lt = ((Es / nat - torch.tensor(b.E_ref, dtype=dt)) ** 2).mean() \
        + ((Ft - torch.tensor(b.F_ref, dtype=dt)) ** 2).sum() / (3 * b.n_atoms) \
        + m.w_S * ((sig - torch.tensor(b.S_ref, dtype=dt)) ** 2).sum() / (9 * S)
    names = [k for k in W if W[k].requires_grad]
    tg = dict(zip(names, torch.autograd.grad(Lt, [W[k] for k in names])))
    np.testing.assert_allclose(aux["stress"], sig.detach().numpy(), rtol=1e-9, atol=1e-14)
    np.testing.assert_allclose(F, Ft.detach().numpy(), rtol=1e-9, atol=1e-12)
    assert loss == pytest.approx(Lt.item(), rel=1e-12)
    for k, v in tg.items():
        v = v.numpy()
        np.testing.assert_allclose(grad[k], v, rtol=0, atol=1e-9 * np.abs(v).max() + 1e-15, err_msg=k)
