"""Pins of the oracle's routing on the evolving edge tokens (logits
(Pc[Z_i] + Pn[Z_j]) + X_e Wr + beta, gates that depend on X_e):

* Wr = 0 gives back the species-pair router: same decisions, energies, forces,
  loss and every other weight gradient;
* the decisions equal a brute-force stable sort of the float64 logits of the
  tokens the forward pass forms;
* forces against central differences of the energy (the gates move with the
  positions through X_e); the loss against central differences in the weights
  (Wr, the species tables, the experts, the radial filter, the embedding) and in
  the positions; every step checked to leave the decisions unchanged; both also
  with self-attention over the neighbourhoods (and its Wqkv, Wo);
* the decision gaps l_(k) - l_(k+1) are those of the sorted logits (reported)."""
import dataclasses

import numpy as np
import pytest

from oracle.model import (Params, build_graph, forces, forward_energy, loss_and_seeds, route_all, training_step,
                          _block_tokens, embed)
from oracle.neighbors import neighbor_list
from paper_2604_15821_amd.synth import _draw_weights, make_batch


def _batch(k=2, seed=3, n_struct=2, wr_scale=1.0, heads=0):
    b = make_batch("tiny", n_struct=n_struct)
    m = dataclasses.replace(b.model, route_feat=1, top_k=k, n_experts=5, n_heads=heads)
    w = _draw_weights(np.random.default_rng(seed), m, 0.0)
    for t in range(m.n_blocks):
        w[f"blocks.{t}.Wr"] = (w[f"blocks.{t}.Wr"] * wr_scale).astype(np.float32)
    return dataclasses.replace(b, model=m, weights=w)


def _state(b, pos, edges, weights=None):
    m = b.model
    P = Params.from_weights(weights if weights is not None else b.weights, m)
    g = build_graph(pos, b.cell, b.offsets, m.r_cut, m.n_rbf, edges)
    rt = route_all(b.species, g, P)
    E, cache = forward_energy(b.species, g, P, rt)
    return P, g, rt, E, cache


def _decisions(rt):
    return [r.eid.copy() for r in rt]


@pytest.mark.parametrize("k", [1, 2])
def test_zero_router_weight_gives_the_species_router(k):
    b = _batch(k=k)
    w0 = dict(b.weights)
    for t in range(b.model.n_blocks):
        w0[f"blocks.{t}.Wr"] = np.zeros_like(w0[f"blocks.{t}.Wr"])
    bf = dataclasses.replace(b, weights=w0)
    base_m = dataclasses.replace(b.model, route_feat=0)
    bs = dataclasses.replace(b, model=base_m, weights={n: v for n, v in w0.items() if not n.endswith(".Wr")})
    l1, E1, F1, g1, a1 = training_step(bf, return_aux=True, positions=True)
    l0, E0, F0, g0, a0 = training_step(bs, return_aux=True, positions=True)
    for r1, r0 in zip(a1["routing"], a0["routing"]):
        assert (r1.eid == r0.eid).all()
    assert l1 == pytest.approx(l0, rel=1e-13)
    np.testing.assert_allclose(E1, E0, rtol=1e-13)
    np.testing.assert_allclose(F1, F0, rtol=0, atol=1e-12 * np.abs(F0).max())
    np.testing.assert_allclose(a1["dLdR"], a0["dLdR"], rtol=0, atol=1e-12 * np.abs(a0["dLdR"]).max())
    for n, v in g0.items():
        np.testing.assert_allclose(g1[n], v, rtol=0, atol=1e-12 * max(np.abs(v).max(), 1e-300), err_msg=n)


def test_decisions_are_the_stable_sort_of_the_logits():
    b = _batch(k=2)
    m = b.model
    edges = neighbor_list(b.pos, b.cell, b.offsets, m.r_cut)
    P, g, rt, E, cache = _state(b, b.pos.astype(np.float64), edges)
    h = cache["h"]
    for t in range(m.n_blocks):
        _, X = _block_tokens(g, P, t, h[t], rt)
        l = ((P.blk(t, "Pc")[b.species[g.ei]] + P.blk(t, "Pn")[b.species[g.ej]]) + X @ P.blk(t, "Wr")) \
            + P.blk(t, "beta")[None, :]
        for e in range(0, l.shape[0], 7):
            order = sorted(range(l.shape[1]), key=lambda x: (-l[e, x], x))
            assert list(rt[t].eid[e]) == order[:m.top_k]
        srt = -np.sort(-l, axis=1)
        assert np.array_equal(rt[t].gap, srt[:, m.top_k - 1] - srt[:, m.top_k])
        scale = 1.0 + np.abs(l).max(1)
        print(f"block {t}: smallest relative gap {(rt[t].gap / scale).min():.2e}, "
              f"{int((rt[t].gap < 1e-5 * scale).sum())} tokens within 1e-5 of a tie")
        assert (rt[t].gap >= 0).all()


@pytest.mark.parametrize("heads", [0, 2])
def test_forces_match_central_differences(heads):
    b = _batch(k=2, heads=heads)
    m = b.model
    edges = neighbor_list(b.pos, b.cell, b.offsets, m.r_cut)
    pos = b.pos.astype(np.float64)
    P, g, rt, E, cache = _state(b, pos, edges)
    F = forces(b.species, g, P, rt, cache)
    h = 1e-5
    rng = np.random.default_rng(2)
    for a in rng.choice(pos.shape[0], 5, replace=False):
        for c in range(3):
            pp, pm = pos.copy(), pos.copy()
            pp[a, c] += h
            pm[a, c] -= h
            sp, sm = _state(b, pp, edges), _state(b, pm, edges)
            for x in (sp, sm):
                for r0, r1 in zip(rt, x[2]):
                    assert (r0.eid == r1.eid).all()
            s = b.offsets.searchsorted(a, side="right") - 1
            fd = -(sp[3][s] - sm[3][s]) / (2 * h)
            assert fd == pytest.approx(F[a, c], rel=1e-6, abs=1e-9 * np.abs(F).max()), (a, c)


@pytest.mark.parametrize("heads", [0, 2])
def test_loss_gradient_matches_central_differences(heads):
    b = _batch(k=2, heads=heads)
    m = b.model
    edges = neighbor_list(b.pos, b.cell, b.offsets, m.r_cut)
    loss, E, F, grad, aux = training_step(b, edges=edges, return_aux=True, positions=True)
    rt0 = aux["routing"]

    def L(weights=None, pos=None):
        P, g, rt, E, cache = _state(b, b.pos.astype(np.float64) if pos is None else pos, edges, weights)
        for r0, r1 in zip(rt0, rt):
            assert (r0.eid == r1.eid).all()
        F = forces(b.species, g, P, rt, cache)
        return loss_and_seeds(E, F, b.E_ref, b.F_ref, g.n_atoms_struct, m.w_E, m.w_F)[0]

    rng = np.random.default_rng(4)
    names = ["blocks.0.Wr", "blocks.1.Wr", "blocks.0.Pc", "blocks.1.Pn", "blocks.0.W1", "blocks.1.W2",
             "blocks.0.W_b", "A", "W_o1"]
    if heads:
        names += ["blocks.0.Wqkv", "blocks.1.Wo"]
    for name in names:
        w = b.weights[name].astype(np.float64)
        scale = np.abs(grad[name]).max()
        for _ in range(3):
            idx = tuple(int(rng.integers(0, n)) for n in w.shape)
            hh = 1e-6 * max(1.0, abs(w[idx]))
            wp, wm = dict(b.weights), dict(b.weights)
            a, c = w.copy(), w.copy()
            a[idx] += hh
            c[idx] -= hh
            wp[name], wm[name] = a, c
            fd = (L(weights=wp) - L(weights=wm)) / (2 * hh)
            assert fd == pytest.approx(grad[name][idx], rel=1e-5, abs=1e-6 * scale), (name, idx)
    pos = b.pos.astype(np.float64)
    dR = aux["dLdR"]
    for a in rng.choice(pos.shape[0], 3, replace=False):
        for c in range(3):
            pp, pm = pos.copy(), pos.copy()
            pp[a, c] += 1e-5
            pm[a, c] -= 1e-5
            fd = (L(pos=pp) - L(pos=pm)) / 2e-5
            assert fd == pytest.approx(dR[a, c], rel=2e-6, abs=2e-7 * np.abs(dR).max()), (a, c)
