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

With the robust loss (paper Sec. "Multi-task training strategies") L is
replaced by (1/S) sum_s W(z_s, tau)^2 L_s over per-structure Huber losses L_s
(``robust_loss_and_seeds``).

With the angular three-body term (``threebody.py``) the edge token gains
the messages of the bond triplets whose first bond is e:
    X_e   = F_e * h_{j(e)} + q_e,   q_e = sum_{tau = (e, .)} MoE3(Z_tau)
and the forces and second-order sweeps carry the angle derivatives.

With the feature-update MoE (paper Sec. "Sparse MoE routing": a second MoE
per block that refines atom features, routed by element type) the block
update becomes
    u_i       = h^t_i + sum_{e : i(e) = i} m_e
    lf_i      = Pf[Z_i] + betaf                      (float32 decision)
    h^{t+1}_i = u_i + sum_c gf_ic W2f_x^T SiLU(W1f_x^T u_i),  x = Kf_i[c]
with the same gating rule as the edge MoE; betaf is fixed like beta.

With the task-aware embedding (paper Sec. "Task-aware feature embedding": a
task (dataset) embedding, charge and spin embeddings and a global embedding
of the element composition) every structure s adds one vector to the
embedding of its atoms:
    h^0_i = A[Z_i] + Tk[task_s] + Qe[charge_s] + Se[spin_s] + c_s Wc,
with c_s the element fractions of s (labels are per-structure indices).

With multi-head self-attention (paper Sec. "Multi-head self-attention",
``attention.py``) the messages of the edges of atom i attend to each other
before they reach the atom:
    u_i = h^t_i + (sum_{e : i(e) = i} u(r_e/r_c) o_e) Wo,
    o = attention over N(i) of m,
with queries, keys and values m [Wq | Wk | Wv] = m Wqkv; the edge envelope
u weighs every edge both as a key (inside the softmax) and as a query (in
the sum), so an edge entering the cutoff changes E smoothly.

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

import math

import numpy as np
import scipy.sparse as sp

from . import attention as attn
from . import threebody as tb
from .basis import bessel_basis, envelope, silu, silu_d1, silu_d2, silu_family
from .neighbors import neighbor_list, reverse_map, triplet_list


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
    three: bool = False
    k3: int = 0
    E3: int = 0
    atom: bool = False
    kf: int = 0
    Ef: int = 0
    heads: int = 0
    r_cut: float = 0.0
    task: bool = False
    route_feat: bool = False

    @classmethod
    def from_weights(cls, weights, model):
        w = {n: np.asarray(v, np.float64) for n, v in weights.items()}
        return cls(w=w, T=model.n_blocks, k=model.top_k, E=model.n_experts, three=bool(model.three_body),
                   k3=model.top_k3, E3=model.n_experts3, atom=bool(model.atom_moe),
                   kf=model.top_k_f, Ef=model.n_experts_f, heads=model.n_heads, r_cut=model.r_cut,
                   task=model.n_tasks > 0, route_feat=bool(getattr(model, "route_feat", 0)))

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
    tri: object = None  # threebody.Triplets when the model has the angular term
    labels: object = None  # (task, charge, spin) per structure for the task-aware embedding


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


def build_graph(batch_pos, cell, offsets, r_cut, n_rbf, edges=None, three=None, labels=None):
    """Neighbour list (unless given as (ei, ej, shift, rowptr)) plus geometry and basis.

    three = (r_cut3, n_legendre) adds the bond triplets and their features;
    labels = (task, charge, spin) per structure feed the task-aware embedding.
    """
    if edges is None:
        edges = neighbor_list(batch_pos, cell, offsets, r_cut)
    ei, ej, shift, rowptr = edges
    d, r, u, sid = edge_geometry(batch_pos, cell, offsets, ei, ej, shift)
    B, dB, _ = bessel_basis(r, r_cut, n_rbf)
    nst = np.diff(np.asarray(offsets, np.int64))
    tri = None
    if three is not None:
        r3, n_l = three
        te, te2, trp = triplet_list(ei, ej, shift, batch_pos, cell, offsets, rowptr, r3)
        tri = tb.triplet_features(te, te2, trp, r, u, r3, n_rbf, n_l)
    return Graph(ei=ei, ej=ej, shift=shift, rowptr=rowptr, d=d, r=r, u=u, B=B, dB=dB,
                 struct_of_atom=sid, n_atoms_struct=nst, tri=tri, labels=labels)


def build_graph_for(batch, edges=None):
    m = batch.model
    three = (m.r_cut3, m.n_legendre) if m.three_body else None
    labels = (batch.task, batch.charge, batch.spin) if m.n_tasks else None
    return build_graph(batch.pos, batch.cell, batch.offsets, m.r_cut, m.n_rbf, edges, three, labels)


def composition(species, g: Graph, n_species):
    """c_s: fraction of the atoms of structure s of each element [S, n_species]."""
    S = g.n_atoms_struct.size
    counts = np.zeros((S, n_species))
    np.add.at(counts, (g.struct_of_atom, species), 1.0)
    return counts / np.maximum(g.n_atoms_struct, 1)[:, None]


def embed(species, g: Graph, P):
    """h^0: the species embedding, plus the per-structure task, charge, spin and
    composition embeddings when the model has them."""
    h = P.w["A"][species]
    if P.task:
        task, charge, spin = g.labels
        c = composition(species, g, P.w["A"].shape[0])
        gs = P.w["Tk"][task] + P.w["Qe"][charge] + P.w["Se"][spin] + c @ P.w["Wc"]
        h = h + gs[g.struct_of_atom]
    return h


# --------------------------------------------------------------------------- routing

@dataclass
class Routing:
    eid: np.ndarray      # [Ne, k] int32 chosen experts (descending logit)
    gate: np.ndarray     # [Ne, k] float64 softmax probability of the chosen expert
    prob: np.ndarray     # [Ne, E] float64 full softmax
    counts: np.ndarray   # [E] int32 tokens per expert
    pos: np.ndarray      # [Ne, k] int32 slot of (e, c) in the expert-grouped order
    inv: np.ndarray      # [Ne*k] int32 flattened (e*k + c) held by each slot
    tri: object = None   # routing of the triplet tokens of the same block (three-body term)
    atom: object = None  # routing of the atom tokens of the feature-update MoE
    Wr: object = None    # routing on the edge tokens: the router's weight [d, E] (gates depend on X)
    gap: object = None   # routing on the edge tokens: l_(k) - l_(k+1) of every token (float64)


def route(species, ei, ej, Pc, Pn, beta, k):
    """Element-type top-k routing of one MoE layer (paper Sec. "Sparse MoE routing").

    Each edge token is routed by the types of its two atoms; the decision is
    taken on float32 logits (Pc[Z_i] + Pn[Z_j]) + beta.  Slots are grouped by
    expert with a stable order on (expert, edge, choice).
    """
    Zi = species[ei]; Zj = species[ej]
    l32 = (np.asarray(Pc, np.float32)[Zi] + np.asarray(Pn, np.float32)[Zj]) + np.asarray(beta, np.float32)[None, :]
    l64 = (np.asarray(Pc, np.float64)[Zi] + np.asarray(Pn, np.float64)[Zj]) + np.asarray(beta, np.float64)[None, :]
    return _route_logits(l32, l64, k)


def route_triplets(species, g, P3a, P3b, P3c, beta3, k3):
    """Routing of triplet tokens by the species of the vertex and of both neighbours:
    logits ((P3a[Z_i] + P3b[Z_j(e)]) + P3c[Z_j(e2)]) + beta3, decided in float32."""
    tri = g.tri
    Zi, Z1, Z2 = species[g.ei[tri.te]], species[g.ej[tri.te]], species[g.ej[tri.te2]]
    f32 = lambda a: np.asarray(a, np.float32)
    f64 = lambda a: np.asarray(a, np.float64)
    l32 = ((f32(P3a)[Zi] + f32(P3b)[Z1]) + f32(P3c)[Z2]) + f32(beta3)[None, :]
    l64 = ((f64(P3a)[Zi] + f64(P3b)[Z1]) + f64(P3c)[Z2]) + f64(beta3)[None, :]
    return _route_logits(l32, l64, k3)


def route_atoms(species, Pf, betaf, kf):
    """Routing of the feature-update MoE: one token per atom, logits Pf[Z_i] + betaf,
    decided in float32 (the element type alone selects the experts)."""
    l32 = np.asarray(Pf, np.float32)[species] + np.asarray(betaf, np.float32)[None, :]
    l64 = np.asarray(Pf, np.float64)[species] + np.asarray(betaf, np.float64)[None, :]
    return _route_logits(l32, l64, kf)


def _route_logits(l32, l64, k):
    """Top-k on float32 logits (lower index first on ties), gates from the float64 softmax."""
    eid = np.argsort(-l32, axis=1, kind="stable")[:, :k].astype(np.int32)
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


def route_features(species, g, Pc, Pn, beta, Wr, X, k):
    """Routing on the evolving edge tokens (the variant of paper Sec. "Sparse MoE routing"
    whose router is a linear layer on the features): logits
        l_e = (Pc[Z_i] + Pn[Z_j]) + X_e Wr + beta
    in float64; top-k descending with the lower index first on ties, gates the softmax
    probabilities of the chosen experts.  The decision is a float64 one here; an fp32
    implementation may differ only where the k-th and (k+1)-th logits are within its
    rounding, which `gap` (l_(k) - l_(k+1), +inf when k = E) exposes."""
    l64 = ((np.asarray(Pc, np.float64)[species[g.ei]] + np.asarray(Pn, np.float64)[species[g.ej]])
           + X @ np.asarray(Wr, np.float64)) + np.asarray(beta, np.float64)[None, :]
    rt = _route_logits(l64, l64, k)
    srt = -np.sort(-l64, axis=1)
    rt.gap = srt[:, k - 1] - srt[:, k] if k < l64.shape[1] else np.full(l64.shape[0], np.inf)
    rt.Wr = np.asarray(Wr, np.float64)
    return rt


def route_all(species, g: Graph, P: Params):
    """Routing of every block (edges, and triplets when the model has the angular term).
    With routing on the edge tokens, block t's decision needs X^t, so the blocks'
    forward pass runs here block by block."""
    if P.route_feat:
        return _route_all_features(species, g, P)
    out = []
    for t in range(P.T):
        rt = route(species, g.ei, g.ej, P.blk(t, "Pc"), P.blk(t, "Pn"), P.blk(t, "beta"), P.k)
        if g.tri is not None:
            rt.tri = route_triplets(species, g, P.blk(t, "P3a"), P.blk(t, "P3b"), P.blk(t, "P3c"),
                                    P.blk(t, "beta3"), P.k3)
        if P.atom:
            rt.atom = route_atoms(species, P.blk(t, "Pf"), P.blk(t, "betaf"), P.kf)
        out.append(rt)
    return out


def _route_all_features(species, g: Graph, P: Params):
    out = []
    N = species.shape[0]
    h = embed(species, g, P)
    for t in range(P.T):
        tri = atom = None
        if g.tri is not None:
            tri = route_triplets(species, g, P.blk(t, "P3a"), P.blk(t, "P3b"), P.blk(t, "P3c"), P.blk(t, "beta3"),
                                 P.k3)
        if P.atom:
            atom = route_atoms(species, P.blk(t, "Pf"), P.blk(t, "betaf"), P.kf)
        # X^t needs this block's triplet routing only
        part = out + [Routing(eid=None, gate=None, prob=None, counts=None, pos=None, inv=None, tri=tri)]
        _, X = _block_tokens(g, P, t, h, part)
        rt = route_features(species, g, P.blk(t, "Pc"), P.blk(t, "Pn"), P.blk(t, "beta"), P.blk(t, "Wr"), X, P.k)
        rt.tri, rt.atom = tri, atom
        out.append(rt)
        m = _moe(rt, P.E, P.blk(t, "W1"), P.blk(t, "W2"), X)
        u = h + _aggregate(g, P, t, m, N)
        h = u + _atom_moe(P, t, out, u)
    return out


# --------------------------------------------------------------------------- forward

def _expert_groups(rt: Routing, E):
    """For each (choice c, expert x): the token rows that send slot c to x."""
    out = []
    for c in range(rt.eid.shape[1]):
        for x in range(E):
            rows = np.nonzero(rt.eid[:, c] == x)[0]
            if rows.size:
                out.append((c, x, rows))
    return out


def _moe(rt, E, W1, W2, X):
    """sum_c g_c W2_x^T SiLU(W1_x^T X) for every token row of X."""
    m = np.zeros((X.shape[0], W2.shape[2]))
    for c, x, rows in _expert_groups(rt, E):
        m[rows] += rt.gate[rows, c][:, None] * (silu(X[rows] @ W1[x]) @ W2[x])
    return m


def _moe_backward(rt, E, W1, W2, X, mbar):
    """Adjoint of the MoE input X given the adjoint mbar of its output.  With routing on
    the tokens (rt.Wr) the gates depend on X too: the gate adjoints <mbar, Y_c> go
    through the softmax Jacobian to the logits, and from them through Wr to X."""
    Xbar = np.zeros_like(X)
    Pg = np.zeros(rt.eid.shape) if rt.Wr is not None else None
    for c, x, rows in _expert_groups(rt, E):
        A = X[rows] @ W1[x]
        Sbar = (rt.gate[rows, c][:, None] * mbar[rows]) @ W2[x].T
        Xbar[rows] += (silu_d1(A) * Sbar) @ W1[x].T
        if Pg is not None:
            Pg[rows, c] = ((silu(A) @ W2[x]) * mbar[rows]).sum(1)
    if Pg is not None:
        Xbar += _logit_adjoint(rt, Pg) @ rt.Wr.T
    return Xbar


def _tri_tokens(g, P, t, h):
    """Z_tau = (G_tau W_a) * h_{j(e2)}; returns (G W_a, h_{j(e2)}, Z)."""
    Zpre = g.tri.G @ P.blk(t, "W_a")
    hj2 = h[g.ej[g.tri.te2]]
    return Zpre, hj2, Zpre * hj2


# --------------------------------------------------------------------------- attention

def _attn_env(g, P):
    """log u(r_e/r_c) of every edge and its derivative in r_e (attention key weights)."""
    u, du, _ = envelope(g.r / P.r_cut)
    return np.log(u), du / (u * P.r_cut)


def _attn_heads(g, P, fn, N, *per_edge):
    """Call fn(i, a, b, cols, slices...) for every (atom, head) neighbourhood; per_edge
    arrays are [Ne, w] with w a multiple of d (column blocks q|k|v, sliced to the head's
    columns) or [Ne] (per-key scalars)."""
    d = P.w["A"].shape[1]
    dh = d // P.heads
    for i in range(N):
        a, b = int(g.rowptr[i]), int(g.rowptr[i + 1])
        if a == b:
            continue
        for hd in range(P.heads):
            cols = np.arange(hd * dh, (hd + 1) * dh)
            args = []
            for x in per_edge:
                if x.ndim == 1:
                    args.append(x[a:b])
                else:
                    args += [x[a:b, j * d + cols] for j in range(x.shape[1] // d)]
            fn(i, a, b, cols, *args)


def _attn_forward(g, P, t, m, lu, N):
    """osum [N, d]: per atom, sum over its edges e of u_e o_e (query weight u_e)."""
    d = m.shape[1]
    QKV = m @ P.blk(t, "Wqkv")
    osum = np.zeros((N, d))

    def fn(i, a, b, cols, q, k, v, l):
        osum[i, cols] = (np.exp(l)[:, None] * attn.forward(q, k, v, l)[0]).sum(0)
    _attn_heads(g, P, fn, N, QKV, lu)
    return osum


def _attn_backward(g, P, t, m, lu, ubar, N):
    """Adjoints of the messages and of log u for the adjoint ubar of u = h + osum Wo."""
    d = m.shape[1]
    QKV = m @ P.blk(t, "Wqkv")
    ob = ubar @ P.blk(t, "Wo").T
    QKVb = np.zeros_like(QKV)
    lub = np.zeros(m.shape[0])

    def fn(i, a, b, cols, q, k, v, l):
        uq = np.exp(l)[:, None]
        o = attn.forward(q, k, v, l)[0]
        qb, kb, vb, lb = attn.backward(q, k, v, l, uq * ob[i, cols][None, :])
        QKVb[a:b, cols], QKVb[a:b, d + cols], QKVb[a:b, 2 * d + cols] = qb, kb, vb
        # log u of an edge enters as key (lb) and through the query weight
        lub[a:b] += lb + uq[:, 0] * (o @ ob[i, cols])
    _attn_heads(g, P, fn, N, QKV, lu)
    return QKVb @ P.blk(t, "Wqkv").T, lub


def _attn_tangent(g, P, t, m, md, lu, rho, N):
    """(osum, osum-dot) for message tangents md and key-weight tangents rho."""
    d = m.shape[1]
    Wqkv = P.blk(t, "Wqkv")
    QKV, QKVd = m @ Wqkv, md @ Wqkv
    osum, osumd = np.zeros((N, d)), np.zeros((N, d))

    def fn(i, a, b, cols, q, k, v, qd, kd, vd, l, r):
        uq = np.exp(l)[:, None]
        o, od = attn.tangent(q, k, v, l, qd, kd, vd, r)
        osum[i, cols] = (uq * o).sum(0)
        osumd[i, cols] = (uq * od + uq * r[:, None] * o).sum(0)
    _attn_heads(g, P, fn, N, QKV, QKVd, lu, rho)
    return osum, osumd


def _attn_reverse(g, P, t, m, md, lu, rho, Pu, Tu, N, bias=None):
    """Reverse sweep of u = h + osum Wo, ud = hd + osumd Wo through the attention:
    returns the adjoints of the messages and of their tangents, dWqkv and dWo.  With
    bias = (Plu, Trho) (arrays [Ne]), also adds the adjoints of every edge's log
    envelope lu and of its tangent rho (as a key inside the softmax and as the query
    weight u = exp(lu))."""
    d = m.shape[1]
    Wqkv, Wo = P.blk(t, "Wqkv"), P.blk(t, "Wo")
    QKV, QKVd = m @ Wqkv, md @ Wqkv
    osum, osumd = _attn_tangent(g, P, t, m, md, lu, rho, N)
    dWo = osum.T @ Pu + osumd.T @ Tu
    Po, To = Pu @ Wo.T, Tu @ Wo.T
    PQ, TQ = np.zeros_like(QKV), np.zeros_like(QKV)

    def fn(i, a, b, cols, q, k, v, qd, kd, vd, l, r):
        # osum = sum u o, osumd = sum u od + u rho o: adjoints of o and od per query
        uq = np.exp(l)[:, None]
        A, B = Po[i, cols][None, :], To[i, cols][None, :]
        res = attn.dual_reverse(q, k, v, l, qd, kd, vd, r, uq * (A + r[:, None] * B), uq * B,
                                key_bias=bias is not None)
        (qb, kb, vb), (qdb, kdb, vdb) = res[0], res[1]
        PQ[a:b, cols], PQ[a:b, d + cols], PQ[a:b, 2 * d + cols] = qb, kb, vb
        TQ[a:b, cols], TQ[a:b, d + cols], TQ[a:b, 2 * d + cols] = qdb, kdb, vdb
        if bias is not None:
            # osum = sum_e u_e o_e, osumd = sum_e u_e (od_e + rho_e o_e), u_e = exp(lu_e)
            o, od = attn.tangent(q, k, v, l, qd, kd, vd, r)
            oA, oB, odB = (o * A).sum(1), (o * B).sum(1), (od * B).sum(1)
            bias[0][a:b] += res[2][0] + uq[:, 0] * (oA + odB + r * oB)
            bias[1][a:b] += res[2][1] + uq[:, 0] * oB
    _attn_heads(g, P, fn, N, QKV, QKVd, lu, rho)
    dWqkv = m.T @ PQ + md.T @ TQ
    return PQ @ Wqkv.T, TQ @ Wqkv.T, dWqkv, dWo


def _aggregate(g, P, t, m, N):
    """Message update of the atoms: sum of the messages, or the attention output."""
    if not P.heads:
        return _seg(g.ei, N, m)
    lu, _ = _attn_env(g, P)
    return _attn_forward(g, P, t, m, lu, N) @ P.blk(t, "Wo")


def _atom_moe(P, t, routing, u):
    """Feature-update MoE output for the atom features u (zero without it)."""
    if not P.atom:
        return np.zeros_like(u)
    return _moe(routing[t].atom, P.Ef, P.blk(t, "W1f"), P.blk(t, "W2f"), u)


def forward_energy(species, g: Graph, P: Params, routing):
    """Forward pass: per-structure energies, the stored atom features h^t and
    the message-updated features u^t of every block."""
    N = species.shape[0]
    Ne = g.ei.shape[0]
    h = embed(species, g, P)
    hs, us = [h], []
    for t in range(P.T):
        F = g.B @ P.blk(t, "W_b")
        X = F * h[g.ej]
        if g.tri is not None:
            _, _, Z = _tri_tokens(g, P, t, h)
            y = _moe(routing[t].tri, P.E3, P.blk(t, "W1a"), P.blk(t, "W2a"), Z)
            X = X + _seg(g.tri.te, Ne, y)
        m = _moe(routing[t], P.E, P.blk(t, "W1"), P.blk(t, "W2"), X)
        u = h + _aggregate(g, P, t, m, N)
        h = u + _atom_moe(P, t, routing, u)
        us.append(u)
        hs.append(h)
    z = h @ P.w["W_o1"]
    eps = silu(z) @ P.w["w_o2"]
    E = _seg(g.struct_of_atom, g.n_atoms_struct.size, eps)
    return E, {"h": hs, "u": us, "z": z, "eps": eps}


def _block_tokens(g, P, t, h, routing):
    """X_e of block t (edge part plus the triplet messages)."""
    F = g.B @ P.blk(t, "W_b")
    X = F * h[g.ej]
    if g.tri is not None:
        _, _, Z = _tri_tokens(g, P, t, h)
        y = _moe(routing[t].tri, P.E3, P.blk(t, "W1a"), P.blk(t, "W2a"), Z)
        X = X + _seg(g.tri.te, g.ei.shape[0], y)
    return F, X


def forces(species, g: Graph, P: Params, routing, cache):
    """Conservative forces F = -dE/dR by one hand-derived reverse sweep."""
    N = species.shape[0]
    G = energy_displacement_gradient(species, g, P, routing, cache)
    dEdR = _seg(g.ej, N, G) - _seg(g.ei, N, G)
    return -dEdR


def stress(g: Graph, G, cell):
    """Stress of every structure from G_e = dE/dd_e (paper Sec. "MatRIS": the stress is
    the strain derivative of the energy over the cell volume).  A strain eps maps every
    displacement d_e to (I + eps) d_e, so dE/deps_ab = sum_e G_e,a d_e,b and
    sigma_s = (1/V_s) sum_{e in s} G_e d_e^T, V_s = |det L_s|."""
    S = g.n_atoms_struct.size
    W = np.zeros((S, 3, 3))
    np.add.at(W, g.struct_of_atom[g.ei], G[:, :, None] * g.d[:, None, :])
    V = np.abs(np.linalg.det(np.asarray(cell, np.float64)))
    return W / V[:, None, None]


def energy_displacement_gradient(species, g: Graph, P: Params, routing, cache):
    """G_e = dE/dd_e of every edge, by one hand-derived reverse sweep."""
    N = species.shape[0]
    Ne = g.ei.shape[0]
    hs, us, z = cache["h"], cache["u"], cache["z"]
    hbar = (silu_d1(z) * P.w["w_o2"][None, :]) @ P.w["W_o1"].T      # dE/dh^T
    rbar = np.zeros(Ne)                                               # dE/dr_e (radial filter)
    Gvec = np.zeros((Ne, 3))                                          # dE/dd_e (triplet features)
    for t in reversed(range(P.T)):
        h = hs[t]
        if P.atom:                                                    # h^{t+1} = u + MoE_f(u)
            hbar = hbar + _moe_backward(routing[t].atom, P.Ef, P.blk(t, "W1f"), P.blk(t, "W2f"), us[t], hbar)
        F, X = _block_tokens(g, P, t, h, routing)
        if P.heads:
            # u = h + attention(m): adjoint of the messages; log u(r) feeds dE/dr
            m = _moe(routing[t], P.E, P.blk(t, "W1"), P.blk(t, "W2"), X)
            lu, dlu = _attn_env(g, P)
            mbar, lub = _attn_backward(g, P, t, m, lu, hbar, N)
            rbar += lub * dlu
        else:
            mbar = hbar[g.ei]
        Xbar = _moe_backward(routing[t], P.E, P.blk(t, "W1"), P.blk(t, "W2"), X, mbar)
        hbar_next = hbar + _seg(g.ej, N, Xbar * F)
        if g.tri is not None:
            Zpre, hj2, Z = _tri_tokens(g, P, t, h)
            Zbar = _moe_backward(routing[t].tri, P.E3, P.blk(t, "W1a"), P.blk(t, "W2a"), Z, Xbar[g.tri.te])
            hbar_next = hbar_next + _seg(g.ej[g.tri.te2], N, Zbar * Zpre)
            Gbar = (Zbar * hj2) @ P.blk(t, "W_a").T
            Gvec += tb.displacement_adjoint(g.tri, g.r, g.u, Gbar, Ne)
        Fbar = Xbar * h[g.ej]
        rbar += ((Fbar @ P.blk(t, "W_b").T) * g.dB).sum(1)
        hbar = hbar_next
    return rbar[:, None] * g.u + Gvec                                 # dE/dd_e


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


def huber2(r, delta):
    """rho(r) = r^2 for |r| <= delta, 2 delta |r| - delta^2 beyond (twice the Huber
    function, so that delta = inf gives the squared error); and rho'(r)."""
    if math.isinf(delta):
        return r * r, 2.0 * r
    a = np.abs(r)
    rho = np.where(a <= delta, r * r, 2.0 * delta * a - delta * delta)
    drho = 2.0 * np.clip(r, -delta, delta)
    return rho, drho


def robust_weight(z, tau):
    """W(z, tau) = exp(-max(z - tau, 0)^2 / 2) and dW/dz: 1 over the normal range
    z <= tau, a smooth (C^1) monotone decay to 0 beyond it."""
    x = np.maximum(z - tau, 0.0)
    W = np.exp(-0.5 * x * x)
    return W, -x * W


def robust_loss_and_seeds(E, F, E_ref, F_ref, offsets, w_E, w_F, delta, tau, task=None, sigma=None,
                          S_ref=None, w_S=0.0):
    """Robust multi-task loss of paper Sec. "Multi-task training strategies" and its
    seeds lam = dL/dE_s, phi = dL/dF_a, psi = dL/dsigma_s.

    L = (1/S) sum_s W(z_s, tau)^2 L_s with the per-structure base loss
        L_s = w_E rho(E_s/n_s - E_ref,s) + w_F/(3 n_s) sum_{a in s, c} rho(F_ac - F_ref,ac)
              + w_S/9 sum_q rho(sigma_sq - S_ref,sq)
    (rho: twice the Huber function of width delta), z_s = (L_s - mu_g)/sd_g standardised
    over the structures of its task g (all structures without tasks; population standard
    deviation; z = 0 where sd_g = 0).  The weights are differentiated like the rest:
    with A_g = sum_{i in g} W_i W'_i L_i and B_g = sum_{i in g} W_i W'_i L_i z_i,
        dL/dL_j = (1/S) [W_j^2 + (2/sd_g)(W_j W'_j L_j - A_g/n_g - z_j B_g/n_g)].
    Readings: the form of W and of rho are not given by the paper (it names a smooth
    monotone soft threshold and an L1 or Huber base loss)."""
    E = np.asarray(E, np.float64)
    F = np.asarray(F, np.float64)
    offsets = np.asarray(offsets, np.int64)
    S = E.shape[0]
    n = np.diff(offsets).astype(np.float64)
    de = E / n - np.asarray(E_ref, np.float64)
    dF = F - np.asarray(F_ref, np.float64)
    rE, dE = huber2(de, delta)
    rF, dFr = huber2(dF, delta)
    sid = np.repeat(np.arange(S), np.diff(offsets))
    L = w_E * rE + w_F * np.bincount(sid, weights=rF.sum(axis=1), minlength=S) / (3.0 * n)
    if w_S:
        ds = np.asarray(sigma, np.float64) - np.asarray(S_ref, np.float64)
        rS, dSr = huber2(ds, delta)
        L = L + w_S * rS.reshape(S, 9).sum(axis=1) / 9.0
    groups = np.zeros(S, np.int64) if task is None else np.asarray(task, np.int64)
    z = np.zeros(S)
    sd = np.zeros(S)
    for gid in np.unique(groups):
        m = groups == gid
        mu = L[m].mean()
        sdg = np.sqrt(((L[m] - mu) ** 2).mean())
        sd[m] = sdg
        if sdg > 0.0:
            z[m] = (L[m] - mu) / sdg
    W, dW = robust_weight(z, tau)
    c = W * W
    for gid in np.unique(groups):
        m = groups == gid
        if sd[m][0] == 0.0:
            continue
        ng = m.sum()
        A = (W * dW * L)[m].sum()
        B = (W * dW * L * z)[m].sum()
        c[m] += 2.0 / sd[m][0] * (W[m] * dW[m] * L[m] - A / ng - z[m] * B / ng)
    c /= S
    loss = (W * W * L).sum() / S
    lam = c * w_E * dE / n
    phi = (c / (3.0 * n) * w_F)[sid][:, None] * dFr
    psi = None
    if w_S:
        psi = (c * w_S / 9.0)[:, None, None] * dSr
    return loss, lam, phi, psi, {"L": L, "z": z, "W": W}


# --------------------------------------------------------------------------- second order

def _gate_tangent(rt, Xd):
    """Tangent of the chosen gates along Xd when the logits are X Wr + const:
    gdot_c = p_x (ldot_x - <p, ldot>), x = eid_c, ldot = Xd Wr.  Also returns ldot."""
    ld = Xd @ rt.Wr
    mu = (rt.prob * ld).sum(1, keepdims=True)
    return rt.gate * (np.take_along_axis(ld, rt.eid.astype(np.int64), 1) - mu), ld


def _moe_tangent(rt, E, W1, W2, X, Xd):
    """MoE output and its tangent for input X and input tangent Xd (with routing on the
    tokens, the gates' own tangent adds gdot_c Y_c)."""
    m = np.zeros((X.shape[0], W2.shape[2]))
    md = np.zeros_like(m)
    gd = _gate_tangent(rt, Xd)[0] if rt.Wr is not None else None
    for c, x, rows in _expert_groups(rt, E):
        A, Ad = X[rows] @ W1[x], Xd[rows] @ W1[x]
        gt = rt.gate[rows, c][:, None]
        s0, s1, _ = silu_family(A)
        Y = s0 @ W2[x]
        m[rows] += gt * Y
        md[rows] += gt * ((s1 * Ad) @ W2[x])
        if gd is not None:
            md[rows] += gd[rows, c][:, None] * Y
    return m, md


def _tri_tangent_tokens(g, P, t, h, hd, Gd):
    """Triplet tokens and their tangents: Z = (G W_a) h_j2, Zd = (Gd W_a) h_j2 + (G W_a) hd_j2."""
    Wa = P.blk(t, "W_a")
    Zpre, Zpred = g.tri.G @ Wa, Gd @ Wa
    j2 = g.ej[g.tri.te2]
    hj2, hdj2 = h[j2], hd[j2]
    return Zpre, Zpred, hj2, hdj2, Zpre * hj2, Zpred * hj2 + Zpre * hdj2


def _block_tangent_tokens(g, P, t, h, hd, Bdot, Gd, routing):
    """X_e, its tangent, and the radial filter with its tangent for block t."""
    Wb = P.blk(t, "W_b")
    F, Fd = g.B @ Wb, Bdot @ Wb
    X = F * h[g.ej]
    Xd = Fd * h[g.ej] + F * hd[g.ej]
    if g.tri is not None:
        Ne = g.ei.shape[0]
        _, _, _, _, Z, Zd = _tri_tangent_tokens(g, P, t, h, hd, Gd)
        y, yd = _moe_tangent(routing[t].tri, P.E3, P.blk(t, "W1a"), P.blk(t, "W2a"), Z, Zd)
        X = X + _seg(g.tri.te, Ne, y)
        Xd = Xd + _seg(g.tri.te, Ne, yd)
    return F, Fd, X, Xd


def stress_loss_and_seed(sigma, S_ref, n_struct_total, w_S):
    """Stress term of the loss, w_S/(9S) sum_s |sigma_s - S_ref,s|_F^2, and its seed
    psi_s = dL/dsigma_s (paper Sec. "Multi-task training strategies" names stress among
    the errors of the base loss; reading: mean-squared error like the other terms)."""
    ds = sigma - np.asarray(S_ref, np.float64)
    return w_S * (ds * ds).sum() / (9.0 * n_struct_total), 2.0 * w_S * ds / (9.0 * n_struct_total)


def displacement_tangent(g: Graph, phi, Psi=None):
    """Tangent of every displacement along the combined direction of the force and
    stress seeds: phi_j - phi_i - Psi_s d_e with Psi_s = psi_s / V_s.  Along it,
    -D E = -D_phi E + sum_s (1/V_s) psi_s : dE/deps_s, so the weight gradient of
    sum_s lam_s E_s - D E is that of the energy + force + stress loss."""
    ddot = phi[g.ej] - phi[g.ei]
    if Psi is not None:
        ddot = ddot - np.einsum("eab,eb->ea", Psi[g.struct_of_atom[g.ei]], g.d)
    return ddot


def energy_tangent(species, g: Graph, P: Params, routing, phi, Psi=None):
    """Tangent forward sweep along positions R + e*phi (and, with Psi, the strain
    direction of the stress seeds).

    Returns (D E_tot, cache) where cache holds per-block primal and
    tangent atom features for the reverse sweep.
    """
    N = species.shape[0]
    ddot = displacement_tangent(g, phi, Psi)                          # d(d_e)/de
    rdot = (ddot * g.u).sum(1)                                         # dr_e/de
    Bdot = g.dB * rdot[:, None]
    Gd = tb.feature_tangent(g.tri, g.r, g.u, ddot) if g.tri is not None else None
    h = embed(species, g, P)
    hd = np.zeros_like(h)
    hs, hds, us, uds = [h], [hd], [], []
    for t in range(P.T):
        F, Fd, X, Xd = _block_tangent_tokens(g, P, t, h, hd, Bdot, Gd, routing)
        m, md = _moe_tangent(routing[t], P.E, P.blk(t, "W1"), P.blk(t, "W2"), X, Xd)
        if P.heads:
            lu, dlu = _attn_env(g, P)
            osum, osumd = _attn_tangent(g, P, t, m, md, lu, dlu * rdot, N)
            u = h + osum @ P.blk(t, "Wo")
            ud = hd + osumd @ P.blk(t, "Wo")
        else:
            u = h + _seg(g.ei, N, m)
            ud = hd + _seg(g.ei, N, md)
        h, hd = u, ud
        if P.atom:
            f, fd = _moe_tangent(routing[t].atom, P.Ef, P.blk(t, "W1f"), P.blk(t, "W2f"), u, ud)
            h, hd = u + f, ud + fd
        us.append(u); uds.append(ud)
        hs.append(h); hds.append(hd)
    z, zd = h @ P.w["W_o1"], hd @ P.w["W_o1"]
    epsd = (silu_d1(z) * zd) @ P.w["w_o2"]
    return epsd.sum(), {"h": hs, "hd": hds, "u": us, "ud": uds, "z": z, "zd": zd, "rdot": rdot, "Bdot": Bdot,
                        "Gd": Gd}


def _moe_reverse(rt, E, W1, W2, X, Xd, Pm, Tm):
    """Reverse sweep of a MoE layer through its primal and tangent outputs.

    Pm, Tm: adjoints of the output and of its tangent.  Returns the adjoints
    of the input and its tangent, the expert weight gradients, the adjoint of
    the router logits and, with routing on the tokens (logits X Wr + const,
    whose gates have the tangent gdot = J(p) Xd Wr), the router weight gradient
    (else None).
    """
    PX = np.zeros_like(X)
    TX = np.zeros_like(X)
    Pg = np.zeros(rt.gate.shape)
    Tg = np.zeros(rt.gate.shape)          # adjoint of the gate tangents
    dW1, dW2 = np.zeros_like(W1), np.zeros_like(W2)
    feat = rt.Wr is not None
    gd, ld = _gate_tangent(rt, Xd) if feat else (None, None)
    for c, x, rows in _expert_groups(rt, E):
        gt = rt.gate[rows, c][:, None]
        A, Ad = X[rows] @ W1[x], Xd[rows] @ W1[x]
        s0, s1, s2 = silu_family(A)
        S, Sd = s0, s1 * Ad
        Y, Yd = S @ W2[x], Sd @ W2[x]
        Pg[rows, c] = (Y * Pm[rows]).sum(1) + (Yd * Tm[rows]).sum(1)
        PY, TY = gt * Pm[rows], gt * Tm[rows]
        if feat:
            # md += gdot Y: adjoints of the gate tangent and of Y through it
            Tg[rows, c] = (Y * Tm[rows]).sum(1)
            PY = PY + gd[rows, c][:, None] * Tm[rows]
        dW2[x] += S.T @ PY + Sd.T @ TY
        PS, TS = PY @ W2[x].T, TY @ W2[x].T
        TAd = s1 * TS
        PA = s1 * PS + s2 * Ad * TS
        dW1[x] += X[rows].T @ PA + Xd[rows].T @ TAd
        PX[rows] += PA @ W1[x].T
        TX[rows] += TAd @ W1[x].T
    Pl = _logit_adjoint(rt, Pg)
    if not feat:
        return PX, TX, dW1, dW2, Pl, None
    # gdot_c = p_x (ld_x - <p, ld>): adjoint of ld is J(p)^T Tg, and of p
    #   Pp_z = Tg~_z (ld_z - <p, ld>) - ld_z sum_c Tg_c p_x(c)   (Tg~: Tg scattered to the chosen experts)
    Tl = _logit_adjoint(rt, Tg)
    Tt = np.zeros(rt.prob.shape)
    np.put_along_axis(Tt, rt.eid.astype(np.int64), Tg, 1)
    mu = (rt.prob * ld).sum(1, keepdims=True)
    Pp = Tt * (ld - mu) - ld * (Tg * rt.gate).sum(1, keepdims=True)
    Pl = Pl + rt.prob * (Pp - (rt.prob * Pp).sum(1, keepdims=True))
    # l = X Wr + const, ld = Xd Wr
    PX += Pl @ rt.Wr.T
    TX += Tl @ rt.Wr.T
    dWr = X.T @ Pl + Xd.T @ Tl
    return PX, TX, dW1, dW2, Pl, dWr


def _logit_adjoint(rt, Pg):
    """Adjoint of the router logits from the adjoints of the chosen gates
    (gates are softmax probabilities: dp_x/dl_y = p_x (delta_xy - p_y))."""
    Pp = np.zeros(rt.prob.shape)
    np.put_along_axis(Pp, rt.eid.astype(np.int64), Pg, 1)
    return rt.prob * (Pp - (rt.prob * Pp).sum(1, keepdims=True))


def weight_gradient(species, g: Graph, P: Params, routing, lam, phi, Psi=None, geo=None):
    """dL/dtheta = d/dtheta [sum_s lam_s E_s - D_phi E] by reverse over the tangent sweep
    (with Psi, the tangent also carries the strain direction of the stress seeds).

    Adjoint names: Pq is the adjoint of primal q, Tq the adjoint of tangent q.  With a
    dict `geo`, the same sweep also leaves there the adjoints of the geometric inputs
    of the bracket: B and Bd = B' rdot [Ne, Nb], with the three-body term G and Gd
    [Nt, L*Nb], with attention the log envelope lu and its tangent rho [Ne].
    """
    N = species.shape[0]
    Ne = g.ei.shape[0]
    _, tc = energy_tangent(species, g, P, routing, phi, Psi)
    hs, hds, z, zd, Bdot, Gd = tc["h"], tc["hd"], tc["z"], tc["zd"], tc["Bdot"], tc["Gd"]
    wo1, wo2 = P.w["W_o1"], P.w["w_o2"]
    grad = {n: np.zeros_like(v) for n, v in P.w.items()}
    S_ = P.w["A"].shape[0]

    if geo is not None:
        geo["B"], geo["Bd"] = np.zeros_like(g.B), np.zeros_like(g.B)
        if g.tri is not None:
            geo["G"], geo["Gd"] = np.zeros_like(g.tri.G), np.zeros_like(g.tri.G)
        if P.heads:
            geo["lu"], geo["rho"] = np.zeros(Ne), np.zeros(Ne)
    lam_atom = lam[g.struct_of_atom][:, None]
    # Psi = sum_i lam_s(i) w_o2.SiLU(z_i) - sum_i w_o2.(SiLU'(z_i) zd_i)
    Pz = lam_atom * silu_d1(z) * wo2 - silu_d2(z) * zd * wo2
    Tz = -silu_d1(z) * wo2
    grad["w_o2"] = (lam_atom * silu(z) - silu_d1(z) * zd).sum(0)
    grad["W_o1"] = hs[-1].T @ Pz + hds[-1].T @ Tz
    Ph, Th = Pz @ wo1.T, Tz @ wo1.T

    for t in reversed(range(P.T)):
        h, hd = hs[t], hds[t]
        rt = routing[t]
        if P.atom:
            # h^{t+1} = u + MoE_f(u), hd^{t+1} = ud + D MoE_f(u) ud: adjoints of u, ud
            u, ud = tc["u"][t], tc["ud"][t]
            PU, TU, dW1f, dW2f, Plf, _ = _moe_reverse(rt.atom, P.Ef, P.blk(t, "W1f"), P.blk(t, "W2f"), u, ud, Ph, Th)
            grad[f"blocks.{t}.W1f"] = dW1f
            grad[f"blocks.{t}.W2f"] = dW2f
            grad[f"blocks.{t}.Pf"] = _seg(species, S_, Plf)
            Ph, Th = Ph + PU, Th + TU
        F, Fd, X, Xd = _block_tangent_tokens(g, P, t, h, hd, Bdot, Gd, routing)
        if P.heads:
            m, md = _moe_tangent(rt, P.E, P.blk(t, "W1"), P.blk(t, "W2"), X, Xd)
            lu, dlu = _attn_env(g, P)
            Pm, Tm, dWqkv, dWo = _attn_reverse(g, P, t, m, md, lu, dlu * tc["rdot"], Ph, Th, N,
                                               bias=None if geo is None else (geo["lu"], geo["rho"]))
            grad[f"blocks.{t}.Wqkv"] = dWqkv
            grad[f"blocks.{t}.Wo"] = dWo
        else:
            Pm, Tm = Ph[g.ei], Th[g.ei]
        PX, TX, dW1, dW2, Pl, dWr = _moe_reverse(rt, P.E, P.blk(t, "W1"), P.blk(t, "W2"), X, Xd, Pm, Tm)
        grad[f"blocks.{t}.W1"] = dW1
        grad[f"blocks.{t}.W2"] = dW2
        if dWr is not None:
            grad[f"blocks.{t}.Wr"] = dWr
        # X = F * h_j (+ q) ;  Xd = Fd * h_j + F * hd_j (+ qd)
        PF = PX * h[g.ej] + TX * hd[g.ej]
        TFd = TX * h[g.ej]
        grad[f"blocks.{t}.W_b"] = g.B.T @ PF + Bdot.T @ TFd
        if geo is not None:
            geo["B"] += PF @ P.blk(t, "W_b").T
            geo["Bd"] += TFd @ P.blk(t, "W_b").T
        Ph_new = Ph + _seg(g.ej, N, PX * F + TX * Fd)
        Th_new = Th + _seg(g.ej, N, TX * F)
        # gates: g_ec = softmax(l_e)[eid_ec];  l_e = Pc[Z_i] + Pn[Z_j] (+ X_e Wr) + beta
        grad[f"blocks.{t}.Pc"] = _seg(species[g.ei], S_, Pl)
        grad[f"blocks.{t}.Pn"] = _seg(species[g.ej], S_, Pl)
        if g.tri is not None:
            tri, rt3 = g.tri, rt.tri
            Zpre, Zpred, hj2, hdj2, Z, Zd = _tri_tangent_tokens(g, P, t, h, hd, Gd)
            # q_e = sum over the triplets of e, so the token adjoints are those of X_e
            PZ, TZ, dW1a, dW2a, Pl3, _ = _moe_reverse(rt3, P.E3, P.blk(t, "W1a"), P.blk(t, "W2a"), Z, Zd,
                                                     PX[tri.te], TX[tri.te])
            grad[f"blocks.{t}.W1a"] = dW1a
            grad[f"blocks.{t}.W2a"] = dW2a
            # Z = Zpre * h_j2 ;  Zd = Zpred * h_j2 + Zpre * hd_j2 ;  Zpre = G W_a, Zpred = Gd W_a
            PZpre = PZ * hj2 + TZ * hdj2
            TZpred = TZ * hj2
            grad[f"blocks.{t}.W_a"] = tri.G.T @ PZpre + Gd.T @ TZpred
            if geo is not None:
                geo["G"] += PZpre @ P.blk(t, "W_a").T
                geo["Gd"] += TZpred @ P.blk(t, "W_a").T
            j2 = g.ej[tri.te2]
            Ph_new = Ph_new + _seg(j2, N, PZ * Zpre + TZ * Zpred)
            Th_new = Th_new + _seg(j2, N, TZ * Zpre)
            grad[f"blocks.{t}.P3a"] = _seg(species[g.ei[tri.te]], S_, Pl3)
            grad[f"blocks.{t}.P3b"] = _seg(species[g.ej[tri.te]], S_, Pl3)
            grad[f"blocks.{t}.P3c"] = _seg(species[j2], S_, Pl3)
        Ph, Th = Ph_new, Th_new
    grad["A"] = _seg(species, P.w["A"].shape[0], Ph)
    if P.task:
        # h0 gains one vector per structure: its adjoint is the sum over the atoms
        task, charge, spin = g.labels
        Pg = _seg(g.struct_of_atom, g.n_atoms_struct.size, Ph)
        grad["Tk"] = _seg(task, P.w["Tk"].shape[0], Pg)
        grad["Qe"] = _seg(charge, P.w["Qe"].shape[0], Pg)
        grad["Se"] = _seg(spin, P.w["Se"].shape[0], Pg)
        grad["Wc"] = composition(species, g, P.w["A"].shape[0]).T @ Pg
    return grad


def position_gradient(species, g: Graph, P: Params, routing, lam, phi, Psi=None, model=None):
    """dL/dR [N, 3] with lam = dL/dE, phi = dL/dF (and Psi = dL/dsigma / V) held fixed.

    Paper Sec. "MatRIS": F = -dE/dR and the stress are derivatives of E, so with the
    seeds frozen the loss varies with the positions like
        Phi = sum_s lam_s E_s - D E,   D E = sum_e G_e . ddot_e,
        ddot_e = phi_j - phi_i - Psi_s d_e,
    because -D E = sum_a phi_a . F_a + sum_s psi_s : sigma_s.  Phi is the bracket whose
    weight gradient weight_gradient takes, so the same reverse sweep through the primal
    and tangent quantities gives the adjoints of its geometric inputs (B, Bd = B' rdot,
    and with the options G, Gd, lu, rho); the chain rule through
        r_e = |d_e|, rdot_e = u_e . ddot_e, Bd = B'(r) rdot  (B'' enters here),
        lu = log u(r / r_c), rho = (d lu / dr) rdot,
    and the triplet features (their second partial derivatives enter through Gd) then
    gives dL/dd_e, and dL/dR_a = sum_{e: j(e) = a} dL/dd_e - sum_{e: i(e) = a} dL/dd_e.
    """
    N = species.shape[0]
    Ne = g.ei.shape[0]
    geo = {}
    grad = weight_gradient(species, g, P, routing, lam, phi, Psi, geo=geo)
    ddot = displacement_tangent(g, phi, Psi)
    rdot = (ddot * g.u).sum(1)
    nb = g.B.shape[1]
    _, dB, d2B = bessel_basis(g.r, P.r_cut, nb)
    adj_r = (geo["B"] * dB).sum(1) + rdot * (geo["Bd"] * d2B).sum(1)
    adj_rdot = (geo["Bd"] * dB).sum(1)
    if P.heads:
        u, du, d2u = envelope(g.r / P.r_cut)
        dlu = du / (u * P.r_cut)                                   # d log u / dr
        d2lu = (d2u / u - (du / u) ** 2) / P.r_cut ** 2
        adj_r = adj_r + geo["lu"] * dlu + geo["rho"] * rdot * d2lu
        adj_rdot = adj_rdot + geo["rho"] * dlu
    # rdot_e = u_e . ddot_e:  d rdot / d d_e = (ddot - rdot u) / r - Psi^T u
    Psi_e = None if Psi is None else Psi[g.struct_of_atom[g.ei]]
    grad_rdot = (ddot - rdot[:, None] * g.u) / g.r[:, None]
    if Psi_e is not None:
        grad_rdot = grad_rdot - np.einsum("eba,eb->ea", Psi_e, g.u)
    adj_d = adj_r[:, None] * g.u + adj_rdot[:, None] * grad_rdot
    if g.tri is not None:
        m = model
        adj_d = adj_d + tb.displacement_adjoint(g.tri, g.r, g.u, geo["G"], Ne)
        adj_d = adj_d + tb.tangent_displacement_adjoint(g.tri, g.r, g.u, ddot, Psi_e, geo["Gd"], m.r_cut3,
                                                        m.n_rbf, m.n_legendre, Ne)
    return _seg(g.ej, N, adj_d) - _seg(g.ei, N, adj_d), grad


# --------------------------------------------------------------------------- one step

def training_step(batch, edges=None, return_aux=False, positions=False):
    """One full training step on a synthetic batch.

    Returns loss, E [S], F [N,3], grad (dict name -> float64 array with the
    weight's shape).  With return_aux, also the graph, the routing and the
    stress [S,3,3].  With w_S > 0 the loss has the stress term.  With positions,
    the aux dict also holds dL/dR [N,3] (position_gradient).
    """
    m = batch.model
    P = Params.from_weights(batch.weights, m)
    g = build_graph_for(batch, edges)
    routing = route_all(batch.species, g, P)
    E, cache = forward_energy(batch.species, g, P, routing)
    G = energy_displacement_gradient(batch.species, g, P, routing, cache)
    N = batch.species.shape[0]
    F = _seg(g.ei, N, G) - _seg(g.ej, N, G)
    sigma = stress(g, G, batch.cell)
    Psi = None
    if getattr(m, "robust", 0):
        loss, lam, phi, psi, _ = robust_loss_and_seeds(
            E, F, batch.E_ref, batch.F_ref, batch.offsets, m.w_E, m.w_F, m.huber_delta, m.robust_tau,
            task=batch.task if m.n_tasks else None, sigma=sigma, S_ref=batch.S_ref, w_S=m.w_S)
        if m.w_S:
            Psi = psi / np.abs(np.linalg.det(np.asarray(batch.cell, np.float64)))[:, None, None]
    else:
        loss, lam, phi = loss_and_seeds(E, F, batch.E_ref, batch.F_ref, g.n_atoms_struct, m.w_E, m.w_F)
        if m.w_S:
            loss_S, psi = stress_loss_and_seed(sigma, batch.S_ref, E.shape[0], m.w_S)
            loss = loss + loss_S
            Psi = psi / np.abs(np.linalg.det(np.asarray(batch.cell, np.float64)))[:, None, None]
    dLdR = None
    if positions:
        dLdR, grad = position_gradient(batch.species, g, P, routing, lam, phi, Psi, model=m)
    else:
        grad = weight_gradient(batch.species, g, P, routing, lam, phi, Psi)
    if return_aux:
        return loss, E, F, grad, {"graph": g, "routing": routing, "lam": lam, "phi": phi, "stress": sigma,
                                  "Psi": Psi, "dLdR": dLdR}
    return loss, E, F, grad


def graph_with_rev(batch):
    m = batch.model
    ei, ej, sh, rp = neighbor_list(batch.pos, batch.cell, batch.offsets, m.r_cut)
    return ei, ej, sh, rp, reverse_map(ei, ej, sh, batch.pos.shape[0])
