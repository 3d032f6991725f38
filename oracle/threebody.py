"""Angular three-body term of the interaction blocks (oracle).

Paper Sec. "MatRIS": pairs of bonds that share an atom define bond angles;
the embedding module turns angles into angle features and every interaction
block has a three-body operation.  The paper prints no formula; the reading
used by the whole build is

  triplet tau = (e, e2)  two distinct edges out of the same centre atom i,
                         both shorter than r3 under the pinned float32 test
  c_tau       = u_e . u_e2                        cosine of the bond angle
  G_tau[l,n]  = P_l(c) B3_n(r_e2) u(r_e / r3)     l < L, n < Nb
                (P_l Legendre; B3 the Bessel basis with cutoff r3, including
                 its own envelope; u the same p = 6 envelope)
  Z_tau       = (G_tau W_a) * h_{j(e2)}
  logits      = ((P3a[Z_i] + P3b[Z_j(e)]) + P3c[Z_j(e2)]) + beta3   (top-k3,
                gates = softmax probabilities of the chosen experts)
  y_tau       = sum_c g3_c W2a_x^T SiLU(W1a_x^T Z_tau)
  q_e         = sum_{tau = (e, .)} y_tau,  added to the edge token X_e.

The envelope on r_e and the basis on r_e2 make each triplet's contribution
vanish with two derivatives when either bond reaches r3.

This module holds the triplet geometry (features and their partial
derivatives with respect to c, r_e and r_e2), the tangent of the features
along a displacement field, the accumulation of a feature adjoint into
per-edge displacement adjoints, and the same for an adjoint of the feature
tangent (which needs the second partial derivatives of the features).  The expert layer itself is evaluated by the
same routines as the edge MoE in ``model.py``.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .basis import bessel_basis, envelope, legendre, legendre2


@dataclass
class Triplets:
    te: np.ndarray       # [Nt] first edge e (its centre atom is the vertex)
    te2: np.ndarray      # [Nt] second edge e2
    trowptr: np.ndarray  # [Ne+1] CSR of the triplets by e
    c: np.ndarray        # [Nt] cos(theta)
    G: np.ndarray        # [Nt, L*Nb] features
    dGdc: np.ndarray     # [Nt, L*Nb] partial derivatives of G
    dGdr1: np.ndarray    # with respect to r_e
    dGdr2: np.ndarray    # with respect to r_e2


def triplet_features(te, te2, trowptr, r, u, r3, n_rbf, n_l):
    """Features of every triplet and their partial derivatives (float64)."""
    u1, u2 = u[te], u[te2]
    r1, r2 = r[te], r[te2]
    c = (u1 * u2).sum(1)
    P, dP = legendre(c, n_l)                         # [Nt, L]
    B3, dB3, _ = bessel_basis(r2, r3, n_rbf)         # [Nt, Nb]
    e3, de3, _ = envelope(r1 / r3)
    de3 = de3 / r3
    nt = te.shape[0]
    outer = lambda a, b: (a[:, :, None] * b[:, None, :]).reshape(nt, a.shape[1] * b.shape[1])
    G = outer(P, B3) * e3[:, None]
    dGdc = outer(dP, B3) * e3[:, None]
    dGdr2 = outer(P, dB3) * e3[:, None]
    dGdr1 = outer(P, B3) * de3[:, None]
    return Triplets(te=te, te2=te2, trowptr=trowptr, c=c, G=G, dGdc=dGdc, dGdr1=dGdr1, dGdr2=dGdr2)


def feature_tangent(tri: Triplets, r, u, ddot):
    """dG/d(eps) for edge displacements d_e + eps * ddot_e."""
    te, te2 = tri.te, tri.te2
    rdot = (u * ddot).sum(1)                                   # d r_e
    udot = (ddot - rdot[:, None] * u) / r[:, None]             # d u_e
    cdot = (udot[te] * u[te2]).sum(1) + (u[te] * udot[te2]).sum(1)
    return tri.dGdc * cdot[:, None] + tri.dGdr1 * rdot[te][:, None] + tri.dGdr2 * rdot[te2][:, None]


def displacement_adjoint(tri: Triplets, r, u, Gbar, n_edges):
    """Adjoint of the edge displacements d_e from an adjoint Gbar of the features.

    c = u_e . u_e2 gives dc/dd_e = (u_e2 - c u_e) / r_e and the symmetric
    term for e2; r depends on d through dr/dd = u.
    """
    te, te2, c = tri.te, tri.te2, tri.c
    ac = (Gbar * tri.dGdc).sum(1)
    a1 = (Gbar * tri.dGdr1).sum(1)
    a2 = (Gbar * tri.dGdr2).sum(1)
    u1, u2, r1, r2 = u[te], u[te2], r[te], r[te2]
    g1 = ac[:, None] * (u2 - c[:, None] * u1) / r1[:, None] + a1[:, None] * u1
    g2 = ac[:, None] * (u1 - c[:, None] * u2) / r2[:, None] + a2[:, None] * u2
    out = np.zeros((n_edges, 3))
    np.add.at(out, te, g1)
    np.add.at(out, te2, g2)
    return out


def tangent_displacement_adjoint(tri: Triplets, r, u, ddot, Psi_e, A, r3, n_rbf, n_l, n_edges):
    """Adjoint of the edge displacements from an adjoint A [Nt, L*Nb] of the feature
    tangent Gd = feature_tangent(tri, r, u, ddot), with ddot_e = phi_j - phi_i - Psi_e d_e
    (Psi_e [Ne, 3, 3] the stress seed over the volume, or None): the gradient in d of

        s = <A, Gd> = g_c cdot + g_1 rdot_e + g_2 rdot_e2,
        g_x = <A, dG/dx>,   rdot = ddot . u,   udot = (ddot - rdot u) / r,
        cdot = udot_e . u_e2 + u_e . udot_e2,

    which needs the second partial derivatives of G = P_l(c) B3_n(r_e2) u(r_e / r3)."""
    te, te2, c = tri.te, tri.te2, tri.c
    u1, u2, r1, r2 = u[te], u[te2], r[te], r[te2]
    dd1, dd2 = ddot[te], ddot[te2]
    nt = te.shape[0]
    P, dP, d2P = legendre2(c, n_l)
    B3, dB3, d2B3 = bessel_basis(r2, r3, n_rbf)
    e3, de3, d2e3 = envelope(r1 / r3)
    de3, d2e3 = de3 / r3, d2e3 / (r3 * r3)
    A3 = A.reshape(nt, n_l, n_rbf)
    pair = lambda a, b: np.einsum("tln,tl,tn->t", A3, a, b)      # <A, a (x) b>
    g_c, g_1, g_2 = pair(dP, B3) * e3, pair(P, B3) * de3, pair(P, dB3) * e3
    g_cc, g_c1, g_c2 = pair(d2P, B3) * e3, pair(dP, B3) * de3, pair(dP, dB3) * e3
    g_11, g_12, g_22 = pair(P, B3) * d2e3, pair(P, dB3) * de3, pair(P, d2B3) * e3
    rd1, rd2 = (dd1 * u1).sum(1), (dd2 * u2).sum(1)
    ud1 = (dd1 - rd1[:, None] * u1) / r1[:, None]
    ud2 = (dd2 - rd2[:, None] * u2) / r2[:, None]
    w1, w2 = (ud1 * u2).sum(1), (u1 * ud2).sum(1)             # cdot = w1 + w2
    cd = w1 + w2
    col = lambda x: x[:, None]
    # Psi^T v for the structure of each triplet (ddot depends on d through -Psi d)
    if Psi_e is not None:
        Ps = Psi_e[te]
        PT = lambda v: np.einsum("tba,tb->ta", Ps, v)
    else:
        PT = lambda v: np.zeros_like(v)
    grad_c1, grad_c2 = (u2 - col(c) * u1) / col(r1), (u1 - col(c) * u2) / col(r2)
    grad_rd1 = ud1 - PT(u1)
    grad_rd2 = ud2 - PT(u2)
    # cdot = w1 + w2, w1 = (ddot_e . u_e2 - rdot_e c) / r_e, w2 = (ddot_e2 . u_e - rdot_e2 c) / r_e2
    grad_w1_d1 = (-PT(u2) - col(c) * grad_rd1 - col(rd1) * grad_c1 - col(w1) * u1) / col(r1)
    grad_w2_d1 = (ud2 - col(w2) * u1) / col(r1)
    grad_w2_d2 = (-PT(u1) - col(c) * grad_rd2 - col(rd2) * grad_c2 - col(w2) * u2) / col(r2)
    grad_w1_d2 = (ud1 - col(w1) * u2) / col(r2)
    a_c = g_cc * cd + g_c1 * rd1 + g_c2 * rd2
    a_1 = g_c1 * cd + g_11 * rd1 + g_12 * rd2
    a_2 = g_c2 * cd + g_12 * rd1 + g_22 * rd2
    t1 = col(a_c) * grad_c1 + col(a_1) * u1 + col(g_c) * (grad_w1_d1 + grad_w2_d1) + col(g_1) * grad_rd1
    t2 = col(a_c) * grad_c2 + col(a_2) * u2 + col(g_c) * (grad_w1_d2 + grad_w2_d2) + col(g_2) * grad_rd2
    out = np.zeros((n_edges, 3))
    np.add.at(out, te, t1)
    np.add.at(out, te2, t2)
    return out
