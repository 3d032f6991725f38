"""Pins of the oracle's neighbourhood self-attention.

Per neighbourhood (oracle/attention.py): the tangent against central
differences of the forward, the backward against the adjoint identity with
those tangents, the dual reverse against central differences of
<Po, o> + <To, o-dot>.  In the model: forces and sampled dL/dW (Wqkv, Wo and
the rest) against central differences; a dimer (one key per neighbourhood)
equals the model without attention whose experts' W2 are W2 Wv Wo; an atom
crossing the cutoff changes the energy continuously with vanishing first
derivative; rotation and permutation invariance; and a torch float64
implementation with forces and weight gradients from autograd."""
import dataclasses

import numpy as np
import pytest

from oracle import attention as attn
from oracle.model import training_step
from paper_2604_15821_amd.synth import Batch, _draw_weights, make_batch


def _inputs(n=7, dh=5, seed=0):
    rng = np.random.default_rng(seed)
    q, k, v, qd, kd, vd = (rng.standard_normal((n, dh)) for _ in range(6))
    lu = np.log(rng.uniform(0.05, 1.0, n))
    rho = rng.standard_normal(n)
    return q, k, v, lu, qd, kd, vd, rho


def test_attention_rows_are_convex_combinations_of_values():
    q, k, v, lu, *_ = _inputs()
    o, p = attn.forward(q, k, v, lu)
    np.testing.assert_allclose(p.sum(1), 1.0, rtol=1e-14)
    assert (p > 0).all()
    # brute force: weights u_l exp(s_el) / sum
    s = q @ k.T / np.sqrt(q.shape[1])
    w = np.exp(lu)[None, :] * np.exp(s)
    np.testing.assert_allclose(o, (w / w.sum(1, keepdims=True)) @ v, rtol=1e-12)


def test_tangent_matches_central_differences():
    q, k, v, lu, qd, kd, vd, rho = _inputs()
    o, od = attn.tangent(q, k, v, lu, qd, kd, vd, rho)
    h = 1e-6
    f = lambda e: attn.forward(q + e * qd, k + e * kd, v + e * vd, lu + e * rho)[0]
    np.testing.assert_allclose(od, (f(h) - f(-h)) / (2 * h), rtol=1e-7, atol=1e-9)


def test_backward_is_the_adjoint_of_the_tangent():
    q, k, v, lu, qd, kd, vd, rho = _inputs(seed=1)
    ob = np.random.default_rng(5).standard_normal(q.shape)
    qb, kb, vb, lub = attn.backward(q, k, v, lu, ob)
    _, od = attn.tangent(q, k, v, lu, qd, kd, vd, rho)
    lhs = (ob * od).sum()
    rhs = (qb * qd).sum() + (kb * kd).sum() + (vb * vd).sum() + (lub * rho).sum()
    assert lhs == pytest.approx(rhs, rel=1e-12)


def test_dual_reverse_matches_central_differences():
    q, k, v, lu, qd, kd, vd, rho = _inputs(seed=2)
    rng = np.random.default_rng(6)
    Po, To = rng.standard_normal(q.shape), rng.standard_normal(q.shape)

    def J(q, k, v, qd, kd, vd):
        o, od = attn.tangent(q, k, v, lu, qd, kd, vd, rho)
        return (Po * o).sum() + (To * od).sum()
    prim, tang = attn.dual_reverse(q, k, v, lu, qd, kd, vd, rho, Po, To)
    args = [q, k, v, qd, kd, vd]
    grads = list(prim) + list(tang)
    h = 1e-6
    for a in range(6):
        for idx in [(0, 0), (3, 2), (6, 4)]:
            ap = [x.copy() for x in args]; ap[a][idx] += h
            am = [x.copy() for x in args]; am[a][idx] -= h
            fd = (J(*ap) - J(*am)) / (2 * h)
            assert fd == pytest.approx(grads[a][idx], rel=1e-6, abs=1e-8), (a, idx)


def _attn_batch(n_struct=2, heads=2, seed=11, **changes):
    b = make_batch("tiny", n_struct=n_struct)
    m = dataclasses.replace(b.model, n_heads=heads, **changes)
    return dataclasses.replace(b, model=m, weights=_draw_weights(np.random.default_rng(seed), m, 0.0))


def test_forces_and_weight_gradient_match_central_differences():
    from oracle.model import Params, build_graph, forces, forward_energy, loss_and_seeds, route_all
    from oracle.neighbors import neighbor_list
    b = _attn_batch()
    m = b.model
    edges = neighbor_list(b.pos, b.cell, b.offsets, m.r_cut)
    loss, E, F, grad, aux = training_step(b, edges=edges, return_aux=True)

    def run(pos, w, routing=None):
        P = Params.from_weights(w, m)
        g = build_graph(pos, b.cell, b.offsets, m.r_cut, m.n_rbf, edges)
        rt = routing if routing is not None else route_all(b.species, g, P)
        E, c = forward_energy(b.species, g, P, rt)
        return E, g, P, c, rt
    pos = b.pos.astype(np.float64)
    rng = np.random.default_rng(0)
    for a in rng.choice(b.n_atoms, 6, replace=False):
        for c in range(3):
            p1 = pos.copy(); p1[a, c] += 1e-5
            p2 = pos.copy(); p2[a, c] -= 1e-5
            fd = -(run(p1, b.weights, aux["routing"])[0].sum() - run(p2, b.weights, aux["routing"])[0].sum()) / 2e-5
            assert abs(fd - F[a, c]) <= 1e-6 * max(1.0, abs(F[a, c]))

    def L(w):
        E, g, P, c, rt = run(b.pos, w)
        for r0, r1 in zip(aux["routing"], rt):
            assert np.array_equal(r0.eid, r1.eid)
        F = forces(b.species, g, P, rt, c)
        return loss_and_seeds(E, F, b.E_ref, b.F_ref, g.n_atoms_struct)[0]
    w64 = {k: v.astype(np.float64) for k, v in b.weights.items()}
    for name in [n for n in w64 if not n.endswith("beta")]:
        W = w64[name]
        picks = [tuple(int(i) for i in np.unravel_index(np.argmax(np.abs(grad[name])), W.shape))]
        picks += [tuple(int(rng.integers(0, s)) for s in W.shape)]
        for idx in picks:
            h = 1e-6 * max(1.0, abs(W[idx]))
            wp = dict(w64); wp[name] = W.copy(); wp[name][idx] += h
            wm = dict(w64); wm[name] = W.copy(); wm[name][idx] -= h
            fd = (L(wp) - L(wm)) / (2 * h)
            scale = max(np.abs(grad[name]).max(), 1e-12)
            assert abs(fd - grad[name][idx]) <= 2e-6 * scale + 1e-9, (name, idx, fd, grad[name][idx])


def _dimer(m, W, r, species=(5, 33)):
    rhat = np.array([0.0, 0.6, 0.8])
    pos = np.array([[9.0, 9.0, 9.0], 9.0 + r * rhat])
    return Batch(pos=pos, cell=np.diag([30.0, 30.0, 30.0])[None].astype(np.float32),
                 species=np.array(species, np.int32), offsets=np.array([0, 2], np.int32),
                 E_ref=np.zeros(1, np.float32), F_ref=np.zeros((2, 3), np.float32), weights=W, model=m)


def test_dimer_equals_the_model_without_attention_with_folded_values():
    """One key per neighbourhood: p = 1 and o_e = m_e Wv, so u = h + u(r/r_c) m Wv Wo; the
    same as the model without attention whose experts' W2 are u(r/r_c) W2 Wv Wo."""
    b = _attn_batch(heads=4)
    m, W = b.model, b.weights
    m0 = dataclasses.replace(m, n_heads=0)
    d = m.d
    W0 = {k: v for k, v in W.items() if not (k.endswith("Wqkv") or k.endswith("Wo"))}
    from oracle.basis import envelope
    for r in (1.7, 3.1):
        ur = envelope(np.array([r / m.r_cut]))[0][0]
        for t in range(m.n_blocks):
            Wv = W[f"blocks.{t}.Wqkv"].astype(np.float64)[:, 2 * d:]
            Wo = W[f"blocks.{t}.Wo"].astype(np.float64)
            W0[f"blocks.{t}.W2"] = ur * W[f"blocks.{t}.W2"].astype(np.float64) @ Wv @ Wo
        l1, E1, F1, g1 = training_step(_dimer(m, W, r))
        l0, E0, F0, g0 = training_step(_dimer(m0, W0, r))
        np.testing.assert_allclose(E1, E0, rtol=1e-12)


def test_energy_is_smooth_when_an_atom_crosses_the_cutoff():
    """A third atom moving through the cutoff of the first: E changes continuously and
    its slope vanishes at r_c (the key weight u(r/r_c) has two vanishing derivatives)."""
    b = _attn_batch(heads=2)
    m, W = b.model, b.weights
    rc = m.r_cut

    def E(x):
        pos = np.array([[10.0, 10.0, 10.0], [11.6, 10.4, 10.0], [10.0 + x, 10.0, 10.0]])
        bb = Batch(pos=pos, cell=np.diag([40.0, 40.0, 40.0])[None].astype(np.float32),
                   species=np.array([3, 17, 50], np.int32), offsets=np.array([0, 3], np.int32),
                   E_ref=np.zeros(1, np.float32), F_ref=np.zeros((3, 3), np.float32), weights=W, model=m)
        return training_step(bb)[1][0]
    # atom 2 is within r_c of atom 0 only for x < r_c (and always within r_c of atom 1).
    # One-sided linear extrapolations to x = r_c agree to O(dx^2) in value and the
    # one-sided slopes to O(dx): E is C^1 across the cutoff.  (A key or query weight
    # without the envelope makes E jump there by O(1).)
    # Both gaps come from the curvature of E alone: they shrink as dx^2 and dx.
    gaps = []
    for dx in (2e-3, 5e-4):
        Em2, Em1, Ep1, Ep2 = E(rc - 2 * dx), E(rc - dx), E(rc + dx), E(rc + 2 * dx)
        gaps.append((abs((2 * Em1 - Em2) - (2 * Ep1 - Ep2)), abs((Em1 - Em2) / dx - (Ep2 - Ep1) / dx)))
    (v1, s1), (v2, s2) = gaps
    assert v1 < 1e-6 and s1 < 5 * 2e-3, gaps
    assert v2 < v1 / 10 and s2 < s1 / 3, gaps
    # the edge matters well inside the cutoff
    assert abs(E(rc - 1.0) - E(rc + 0.5)) > 1e-3


def test_rotation_and_permutation_invariance():
    b = _attn_batch(n_struct=2)
    l0, E0, F0, g0 = training_step(b)
    rng = np.random.default_rng(4)
    qm, rr = np.linalg.qr(rng.standard_normal((3, 3)))
    qm = qm * np.sign(np.diag(rr))
    b2 = dataclasses.replace(b, pos=b.pos.astype(np.float64) @ qm.T, cell=b.cell.astype(np.float64) @ qm.T)
    l1, E1, F1, g1 = training_step(b2)
    np.testing.assert_allclose(E1, E0, rtol=1e-11)
    np.testing.assert_allclose(F1, F0 @ qm.T, rtol=1e-8, atol=1e-10)
    perm = np.concatenate([b.offsets[s] + rng.permutation(b.offsets[s + 1] - b.offsets[s])
                           for s in range(b.n_struct)])
    b3 = dataclasses.replace(b, pos=b.pos[perm], species=b.species[perm], F_ref=b.F_ref[perm])
    l3, E3, F3, g3 = training_step(b3)
    np.testing.assert_allclose(E3, E0, rtol=1e-12)
    np.testing.assert_allclose(F3, F0[perm], rtol=1e-9, atol=1e-12)
    for k in g0:
        np.testing.assert_allclose(g3[k], g0[k], rtol=1e-9, atol=1e-12 * max(1.0, np.abs(g0[k]).max()))


torch = pytest.importorskip("torch")


def test_oracle_matches_torch_double_backward_with_attention():
    b = _attn_batch(n_struct=2, heads=4)
    loss, E, F, grad, aux = training_step(b, return_aux=True)
    g, rts, m = aux["graph"], aux["routing"], b.model
    dt = torch.float64
    pos = torch.tensor(b.pos, dtype=dt, requires_grad=True)
    cell = torch.tensor(b.cell, dtype=dt)
    W = {k: torch.tensor(v, dtype=dt, requires_grad=not k.endswith("beta")) for k, v in b.weights.items()}
    Z = torch.tensor(b.species, dtype=torch.long)
    ei, ej = torch.tensor(g.ei, dtype=torch.long), torch.tensor(g.ej, dtype=torch.long)
    sid = torch.tensor(g.struct_of_atom, dtype=torch.long)
    d = pos[ej] - pos[ei] + torch.einsum("ek,ekc->ec", torch.tensor(g.shift, dtype=dt), cell[sid[ei]])
    r = torch.sqrt((d * d).sum(1))
    n = torch.arange(1, m.n_rbf + 1, dtype=dt)
    x = r / m.r_cut
    u = 1 - 28 * x ** 6 + 48 * x ** 7 - 21 * x ** 8
    B = (2.0 / m.r_cut) ** 0.5 * torch.sin(n[None] * np.pi * r[:, None] / m.r_cut) / r[:, None] * u[:, None]
    N, D, H = b.n_atoms, m.d, m.n_heads
    dh = D // H
    h = W["A"][Z]
    rowptr = g.rowptr
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
        QKV = msg @ W[p + "Wqkv"]
        osum = []
        for i in range(N):
            a, bnd = int(rowptr[i]), int(rowptr[i + 1])
            if a == bnd:
                osum.append(torch.zeros(D, dtype=dt))
                continue
            heads = []
            for hd in range(H):
                q = QKV[a:bnd, hd * dh:(hd + 1) * dh]
                k = QKV[a:bnd, D + hd * dh:D + (hd + 1) * dh]
                v = QKV[a:bnd, 2 * D + hd * dh:2 * D + (hd + 1) * dh]
                wts = torch.softmax(q @ k.T / dh ** 0.5 + torch.log(u[a:bnd])[None, :], dim=1)
                heads.append((u[a:bnd][:, None] * (wts @ v)).sum(0))
            osum.append(torch.cat(heads))
        h = h + torch.stack(osum) @ W[p + "Wo"]
    eps = torch.nn.functional.silu(h @ W["W_o1"]) @ W["w_o2"]
    Es = torch.zeros(b.n_struct, dtype=dt).index_add(0, sid, eps)
    Ft = -torch.autograd.grad(Es.sum(), pos, create_graph=True)[0]
    nat = torch.tensor(np.diff(b.offsets), dtype=dt)
    Lt = ((Es / nat - torch.tensor(b.E_ref, dtype=dt)) ** 2).mean() \
        + ((Ft - torch.tensor(b.F_ref, dtype=dt)) ** 2).sum() / (3 * N)
    names = [k for k in W if W[k].requires_grad]
    tg = dict(zip(names, torch.autograd.grad(Lt, [W[k] for k in names])))
    assert loss == pytest.approx(Lt.item(), rel=1e-12)
    np.testing.assert_allclose(E, Es.detach().numpy(), rtol=1e-12)
    np.testing.assert_allclose(F, Ft.detach().numpy(), rtol=1e-9, atol=1e-12)
    for k, v in tg.items():
        v = v.numpy()
        np.testing.assert_allclose(grad[k], v, rtol=0, atol=1e-9 * np.abs(v).max() + 1e-15, err_msg=k)
