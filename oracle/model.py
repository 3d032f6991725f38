"""Energy, forces, loss and weight gradients of the MoE potential (oracle).

Model (paper Sec. "MatRIS" and Sec. "Algorithmic innovation / sparse MoE
routing"; the paper prints no equations, so the reading below is the one the
whole build follows).  All arithmetic is float64 on float32 inputs widened
exactly; only the two integer decisions (neighbour inclusion, top-k) are
taken in float32 so that both sides take them identically.

  h^0_i   = A[Z_i]                                   species embedding
  block t = 0..T-1:
    F_e   = B(r_e) W_b                               radial filter   [d]
    X_e   = F_e * h_{j(e)}                           edge token      [d]
    l_e   = (Pc[Z_i] + Pn[Z_j]) + beta               router logits   [E]
            (float32 for the top-k decision; the decision depends on
             element types only, as the paper's routing does)
    K_e   = top-k of l_e (descending; lower index wins ties)
    p_e   = softmax(l_e) over all E experts; gate of slot c: g_ec = p_e[K_e[c]]
    m_e   = sum_c g_ec * W2_x^T SiLU(W1_x^T X_e),  x = K_e[c]
    h^{t+1}_i = h^t_i + sum_{e : i(e) = i} m_e
  eps_i   = w_o2 . SiLU(W_o1^T h^T_i)                per-atom energy
  E_s     = sum_{i in s} eps_i
  F_a     = -dE/dR_a                                 conservative forces
  L       = w_E/S sum_s (E_s/n_s - E_ref,s)^2 + w_F/(3N) sum_a |F_a - F_ref,a|^2

beta is a fixed routing bias (it receives no gradient).

Second order (paper Sec. "Runtime for multi-phase double-backward
execution": the force loss needs derivatives of F with respect to the
weights).  With lam_s = dL/dE_s and phi_a = dL/dF_a held fixed,

  dL/dtheta = d/dtheta [ sum_s lam_s E_s - D_phi E ],
  D_phi E   = d/de  E_tot(R + e phi) |_{e=0}   (directional derivative),

because F = -dE/dR.  This oracle evaluates D_phi E with a tangent (dual
number) forward sweep and then takes one reverse sweep of the bracket through
both the primal and the tangent quantities.  That is a different derivation
from the paper's four-phase reverse-over-reverse schedule, which the HIP
path follows, so a mistake in either derivation does not cancel.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import scipy.sparse as sp

from .basis import bessel_basis, silu, silu_d1, silu_d2, silu_family
from .neighbors import neighbor_list, reverse_map


# --------------------------------------------------------------------------- helpers

def _seg(index, n, values):
    """sum over rows of `values` grouped by `index` -> [n, ...] (library sparse matmul)."""
    m = index.shape[0]
    mat = sp.csr_matrix((np.ones(m), (np.asarray(index, np.int64), np.arange(m))), shape=(n, m))
    return mat @ values


@dataclass
class Params:
    """float64 copies of the weight tensors, by name."""

    w: dict
    T: int
    k: int
    E: int

    @classmethod
    def from_weights(cls, weights, model):
        w = {n: np.asarray(v, np.float64) for n, v in weights.items()}
        return cls(w=w, T=model.n_blocks, k=model.top_k, E=model.n_experts)

    def blk(self, t, name):
        return self.w[f"blocks.{t}.{name}"]


@dataclass
class Graph:
    """Edges and their geometry for one batch (float64 geometry)."""

    ei: np.ndarray
    ej: np.ndarray
    shift: np.ndarray
    rowptr: np.ndarray
    d: np.ndarray       # [Ne, 3] displacement X_j + n.L - X_i
    r: np.ndarray       # [Ne]
    u: np.ndarray       # [Ne, 3] unit vector d / r
    B: np.ndarray       # [Ne, Nb]
    dB: np.ndarray      # [Ne, Nb]
    struct_of_atom: np.ndarray
    n_atoms_struct: np.ndarray


def edge_geometry(pos, cell, offsets, ei, ej, shift):
    """float64 displacement d_e = X_j + n.L - X_i, distance and unit vector."""
    pos = np.asarray(pos, np.float64)
    cell = np.asarray(cell, np.float64)
    N = pos.shape[0]
    sid = np.zeros(N, np.int64)
    for s in range(cell.shape[0]):
        sid[int(offsets[s]):int(offsets[s + 1])] = s
    L = cell[sid[ei]]
    n = shift.astype(np.float64)
    d = pos[ej] - pos[ei] + np.einsum("ek,ekc->ec", n, L)
    r = np.sqrt((d * d).sum(1))
    return d, r, d / r[:, None], sid


def build_graph(batch_pos, cell, offsets, r_cut, n_rbf, edges=None):
    """Neighbour list (unless given as (ei, ej, shift, rowptr)) plus geometry and basis."""
    if edges is None:
        edges = neighbor_list(batch_pos, cell, offsets, r_cut)
    ei, ej, shift, rowptr = edges
    d, r, u, sid = edge_geometry(batch_pos, cell, offsets, ei, ej, shift)
    B, dB, _ = bessel_basis(r, r_cut, n_rbf)
    nst = np.diff(np.asarray(offsets, np.int64))
    return Graph(ei=ei, ej=ej, shift=shift, rowptr=rowptr, d=d, r=r, u=u, B=B, dB=dB,
                 struct_of_atom=sid, n_atoms_struct=nst)


# --------------------------------------------------------------------------- routing

@dataclass
class Routing:
    eid: np.ndarray      # [Ne, k] int32 chosen experts (descending logit)
    gate: np.ndarray     # [Ne, k] float64 softmax probability of the chosen expert
    prob: np.ndarray     # [Ne, E] float64 full softmax
    counts: np.ndarray   # [E] int32 tokens per expert
    pos: np.ndarray      # [Ne, k] int32 slot of (e, c) in the expert-grouped order
    inv: np.ndarray      # [Ne*k] int32 flattened (e*k + c) held by each slot


def route(species, ei, ej, Pc, Pn, beta, k):
    """Element-type top-k routing of one MoE layer (paper Sec. "Sparse MoE routing").

    Each edge token is routed by the types of its two atoms; the decision is
    taken on float32 logits (Pc[Z_i] + Pn[Z_j]) + beta.  Slots are grouped by
    expert with a stable order on (expert, edge, choice).
    """
    Zi = species[ei]; Zj = species[ej]
    l32 = (np.asarray(Pc, np.float32)[Zi] + np.asarray(Pn, np.float32)[Zj]) + np.asarray(beta, np.float32)[None, :]
    eid = np.argsort(-l32, axis=1, kind="stable")[:, :k].astype(np.int32)
    l64 = (np.asarray(Pc, np.float64)[Zi] + np.asarray(Pn, np.float64)[Zj]) + np.asarray(beta, np.float64)[None, :]
    l64 = l64 - l64.max(1, keepdims=True)
    ex = np.exp(l64)
    prob = ex / ex.sum(1, keepdims=True)
    gate = np.take_along_axis(prob, eid.astype(np.int64), 1)
    E = prob.shape[1]
    flat = eid.reshape(-1)
    inv = np.argsort(flat, kind="stable").astype(np.int32)
    pos = np.empty_like(inv)
    pos[inv] = np.arange(inv.size, dtype=np.int32)
    counts = np.bincount(flat, minlength=E).astype(np.int32)
    return Routing(eid=eid, gate=gate, prob=prob, counts=counts, pos=pos.reshape(eid.shape), inv=inv)


def route_all(species, g: Graph, P: Params):
    return [route(species, g.ei, g.ej, P.blk(t, "Pc"), P.blk(t, "Pn"), P.blk(t, "beta"), P.k)
            for t in range(P.T)]


# --------------------------------------------------------------------------- forward

def _expert_groups(rt: Routing, E):
    """For each (choice c, expert x): the edge rows that send slot c to x."""
    out = []
    for c in range(rt.eid.shape[1]):
        for x in range(E):
            rows = np.nonzero(rt.eid[:, c] == x)[0]
            if rows.size:
                out.append((c, x, rows))
    return out


def forward_energy(species, g: Graph, P: Params, routing):
    """Forward pass: per-structure energies and the stored atom features h^t."""
    N = species.shape[0]
    h = P.w["A"][species]
    hs = [h]
    for t in range(P.T):
        F = g.B @ P.blk(t, "W_b")
        X = F * h[g.ej]
        m = np.zeros_like(X)
        W1, W2 = P.blk(t, "W1"), P.blk(t, "W2")
        for c, x, rows in _expert_groups(routing[t], P.E):
            Y = silu(X[rows] @ W1[x]) @ W2[x]
            m[rows] += routing[t].gate[rows, c][:, None] * Y
        h = h + _seg(g.ei, N, m)
        hs.append(h)
    z = h @ P.w["W_o1"]
    eps = silu(z) @ P.w["w_o2"]
    E = _seg(g.struct_of_atom, g.n_atoms_struct.size, eps)
    return E, {"h": hs, "z": z, "eps": eps}


def forces(species, g: Graph, P: Params, routing, cache):
    """Conservative forces F = -dE/dR by one hand-derived reverse sweep."""
    N = species.shape[0]
    hs, z = cache["h"], cache["z"]
    hbar = (silu_d1(z) * P.w["w_o2"][None, :]) @ P.w["W_o1"].T      # dE/dh^T
    rbar = np.zeros(g.r.shape[0])                                     # dE/dr_e
    for t in reversed(range(P.T)):
        h = hs[t]
        F = g.B @ P.blk(t, "W_b")
        X = F * h[g.ej]
        mbar = hbar[g.ei]
        Xbar = np.zeros_like(X)
        W1, W2 = P.blk(t, "W1"), P.blk(t, "W2")
        rt = routing[t]
        for c, x, rows in _expert_groups(rt, P.E):
            A = X[rows] @ W1[x]
            Sbar = (rt.gate[rows, c][:, None] * mbar[rows]) @ W2[x].T
            Xbar[rows] += (silu_d1(A) * Sbar) @ W1[x].T
        Fbar = Xbar * h[g.ej]
        rbar += ((Fbar @ P.blk(t, "W_b").T) * g.dB).sum(1)
        hbar = hbar + _seg(g.ej, N, Xbar * F)
    G = rbar[:, None] * g.u                                           # dE/dd_e
    dEdR = _seg(g.ej, N, G) - _seg(g.ei, N, G)
    return -dEdR


def loss_and_seeds(E, F, E_ref, F_ref, n_atoms_struct, w_E=1.0, w_F=1.0):
    """Energy+force loss and its adjoint seeds lam = dL/dE_s, phi = dL/dF_a.

    Paper Sec. "Multi-task training strategies": the base loss combines
    energy and force errors.  Reading: mean-squared errors, energy per atom.
    """
    S = E.shape[0]
    N = F.shape[0]
    n = n_atoms_struct.astype(np.float64)
    de = E / n - np.asarray(E_ref, np.float64)
    dF = F - np.asarray(F_ref, np.float64)
    loss = w_E * (de * de).sum() / S + w_F * (dF * dF).sum() / (3.0 * N)
    lam = 2.0 * w_E * de / (S * n)
    phi = 2.0 * w_F * dF / (3.0 * N)
    return loss, lam, phi


# --------------------------------------------------------------------------- second order

def energy_tangent(species, g: Graph, P: Params, routing, phi):
    """Tangent forward sweep along positions R + e*phi.

    Returns (D_phi E_tot, cache) where cache holds per-block primal and
    tangent atom features for the reverse sweep.
    """
    N = species.shape[0]
    rdot = ((phi[g.ej] - phi[g.ei]) * g.u).sum(1)                      # dr_e/de
    Bdot = g.dB * rdot[:, None]
    h = P.w["A"][species]
    hd = np.zeros_like(h)
    hs, hds = [h], [hd]
    for t in range(P.T):
        Wb = P.blk(t, "W_b")
        F, Fd = g.B @ Wb, Bdot @ Wb
        X = F * h[g.ej]
        Xd = Fd * h[g.ej] + F * hd[g.ej]
        m = np.zeros_like(X); md = np.zeros_like(X)
        W1, W2 = P.blk(t, "W1"), P.blk(t, "W2")
        for c, x, rows in _expert_groups(routing[t], P.E):
            A, Ad = X[rows] @ W1[x], Xd[rows] @ W1[x]
            gt = routing[t].gate[rows, c][:, None]
            s0, s1, _ = silu_family(A)
            m[rows] += gt * (s0 @ W2[x])
            md[rows] += gt * ((s1 * Ad) @ W2[x])
        h = h + _seg(g.ei, N, m)
        hd = hd + _seg(g.ei, N, md)
        hs.append(h); hds.append(hd)
    z, zd = h @ P.w["W_o1"], hd @ P.w["W_o1"]
    epsd = (silu_d1(z) * zd) @ P.w["w_o2"]
    return epsd.sum(), {"h": hs, "hd": hds, "z": z, "zd": zd, "rdot": rdot, "Bdot": Bdot}


def weight_gradient(species, g: Graph, P: Params, routing, lam, phi):
    """dL/dtheta = d/dtheta [sum_s lam_s E_s - D_phi E] by reverse over the tangent sweep.

    Adjoint names: Pq is the adjoint of primal q, Tq the adjoint of tangent q.
    """
    N = species.shape[0]
    _, tc = energy_tangent(species, g, P, routing, phi)
    hs, hds, z, zd, Bdot = tc["h"], tc["hd"], tc["z"], tc["zd"], tc["Bdot"]
    wo1, wo2 = P.w["W_o1"], P.w["w_o2"]
    grad = {n: np.zeros_like(v) for n, v in P.w.items()}

    lam_atom = lam[g.struct_of_atom][:, None]
    # Psi = sum_i lam_s(i) w_o2.SiLU(z_i) - sum_i w_o2.(SiLU'(z_i) zd_i)
    Pz = lam_atom * silu_d1(z) * wo2 - silu_d2(z) * zd * wo2
    Tz = -silu_d1(z) * wo2
    grad["w_o2"] = (lam_atom * silu(z) - silu_d1(z) * zd).sum(0)
    grad["W_o1"] = hs[-1].T @ Pz + hds[-1].T @ Tz
    Ph, Th = Pz @ wo1.T, Tz @ wo1.T

    for t in reversed(range(P.T)):
        h, hd = hs[t], hds[t]
        Wb = P.blk(t, "W_b")
        F, Fd = g.B @ Wb, Bdot @ Wb
        X = F * h[g.ej]
        Xd = Fd * h[g.ej] + F * hd[g.ej]
        Pm, Tm = Ph[g.ei], Th[g.ei]
        PX = np.zeros_like(X); TX = np.zeros_like(X)
        rt = routing[t]
        Pg = np.zeros(rt.gate.shape)
        W1, W2 = P.blk(t, "W1"), P.blk(t, "W2")
        dW1, dW2 = np.zeros_like(W1), np.zeros_like(W2)
        for c, x, rows in _expert_groups(rt, P.E):
            gt = rt.gate[rows, c][:, None]
            A, Ad = X[rows] @ W1[x], Xd[rows] @ W1[x]
            s0, s1, s2 = silu_family(A)
            S, Sd = s0, s1 * Ad
            Y, Yd = S @ W2[x], Sd @ W2[x]
            Pg[rows, c] = (Y * Pm[rows]).sum(1) + (Yd * Tm[rows]).sum(1)
            PY, TY = gt * Pm[rows], gt * Tm[rows]
            dW2[x] += S.T @ PY + Sd.T @ TY
            PS, TS = PY @ W2[x].T, TY @ W2[x].T
            TAd = s1 * TS
            PA = s1 * PS + s2 * Ad * TS
            dW1[x] += X[rows].T @ PA + Xd[rows].T @ TAd
            PX[rows] += PA @ W1[x].T
            TX[rows] += TAd @ W1[x].T
        grad[f"blocks.{t}.W1"] = dW1
        grad[f"blocks.{t}.W2"] = dW2
        # X = F * h_j ;  Xd = Fd * h_j + F * hd_j
        PF = PX * h[g.ej] + TX * hd[g.ej]
        TFd = TX * h[g.ej]
        grad[f"blocks.{t}.W_b"] = g.B.T @ PF + Bdot.T @ TFd
        Ph = Ph + _seg(g.ej, N, PX * F + TX * Fd)
        Th = Th + _seg(g.ej, N, TX * F)
        # gates: g_ec = softmax(l_e)[eid_ec];  l_e = Pc[Z_i] + Pn[Z_j] + beta
        Pp = np.zeros(rt.prob.shape)
        np.put_along_axis(Pp, rt.eid.astype(np.int64), Pg, 1)
        Pl = rt.prob * (Pp - (rt.prob * Pp).sum(1, keepdims=True))
        S_ = P.w["A"].shape[0]
        grad[f"blocks.{t}.Pc"] = _seg(species[g.ei], S_, Pl)
        grad[f"blocks.{t}.Pn"] = _seg(species[g.ej], S_, Pl)
    grad["A"] = _seg(species, P.w["A"].shape[0], Ph)
    return grad


# --------------------------------------------------------------------------- one step

def training_step(batch, edges=None, return_aux=False):
    """One full training step on a synthetic batch.

    Returns loss, E [S], F [N,3], grad (dict name -> float64 array with the
    weight's shape).  With return_aux, also the graph and routing.
    """
    m = batch.model
    if m.three_body:
        raise NotImplementedError("three-body term: see oracle.threebody")
    P = Params.from_weights(batch.weights, m)
    g = build_graph(batch.pos, batch.cell, batch.offsets, m.r_cut, m.n_rbf, edges)
    routing = route_all(batch.species, g, P)
    E, cache = forward_energy(batch.species, g, P, routing)
    F = forces(batch.species, g, P, routing, cache)
    loss, lam, phi = loss_and_seeds(E, F, batch.E_ref, batch.F_ref, g.n_atoms_struct, m.w_E, m.w_F)
    grad = weight_gradient(batch.species, g, P, routing, lam, phi)
    if return_aux:
        return loss, E, F, grad, {"graph": g, "routing": routing, "lam": lam, "phi": phi}
    return loss, E, F, grad


def graph_with_rev(batch):
    m = batch.model
    ei, ej, sh, rp = neighbor_list(batch.pos, batch.cell, batch.offsets, m.r_cut)
    return ei, ej, sh, rp, reverse_map(ei, ej, sh, batch.pos.shape[0])
