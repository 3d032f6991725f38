"""Multi-head self-attention over one atom's neighbourhood (oracle).

Test infrastructure: used only by the tests, the smoke check and the CPU
baseline of the benchmark; it shares no code with the HIP path.

Paper Sec. "Multi-head self-attention": MatRIS-MoE replaces its separable
attention by multi-head self-attention whose cost at a fixed cutoff is
O(m d sum_i |N(i)|^2), i.e. every edge of a neighbourhood attends to every
edge of the same neighbourhood.  Reading used here (the paper gives no
formula): the tokens of atom i are the messages m_e of its edges e in N(i);
head a of width dh = d/m uses columns [a dh, (a+1) dh) of
    q = m Wq,  k = m Wk,  v = m Wv;
the weights are a softmax over the keys of the scores q.k / sqrt(dh) with
the edge envelope u(r_e'/r_c) as a multiplicative weight,
    p_ee' = u_e' exp(s_ee') / sum_l u_l exp(s_el),
and o_e = sum_e' p_ee' v_e'.  The atom receives sum_e u_e o_e (model.py):
the envelope weighs every edge as a key and as a query, so an edge entering
the cutoff (u = 0 with two vanishing derivatives) changes nothing abruptly.

The functions below act on one neighbourhood and one head (arrays [n, dh]);
lu = log u of the keys, rho = tangent of lu.  Each follows the plain
definition of the quantity it returns:
  forward      o = p v
  tangent      o-dot for input tangents (q, k, v, lu)-dot
  backward     adjoints of q, k, v and lu for an adjoint of o
  dual_reverse adjoints of the primal and tangent inputs for adjoints of
               o and of o-dot (the reverse sweep through both), optionally
               including the key weights lu and their tangents rho.
"""
from __future__ import annotations

import numpy as np


def _softmax(z):
    z = z - z.max(1, keepdims=True)
    e = np.exp(z)
    return e / e.sum(1, keepdims=True)


def weights(q, k, lu):
    """p [n, n]: softmax over keys of q.k/sqrt(dh) + log u(key)."""
    return _softmax(q @ k.T / np.sqrt(q.shape[1]) + lu[None, :])


def forward(q, k, v, lu):
    p = weights(q, k, lu)
    return p @ v, p


def tangent(q, k, v, lu, qd, kd, vd, rho):
    """(o, o-dot): p-dot = p * (z-dot - <p, z-dot>), z-dot = (qd k^T + q kd^T)/sqrt(dh) + rho."""
    c = np.sqrt(q.shape[1])
    p = weights(q, k, lu)
    zd = (qd @ k.T + q @ kd.T) / c + rho[None, :]
    pd = p * (zd - (p * zd).sum(1, keepdims=True))
    return p @ v, pd @ v + p @ vd


def backward(q, k, v, lu, ob):
    """Adjoints (qb, kb, vb, lub) of the inputs for the adjoint ob [n, dh] of o."""
    c = np.sqrt(q.shape[1])
    p = weights(q, k, lu)
    pb = ob @ v.T
    zb = p * (pb - (p * pb).sum(1, keepdims=True))
    return zb @ k / c, zb.T @ q / c, p.T @ ob, zb.sum(0)


def dual_reverse(q, k, v, lu, qd, kd, vd, rho, Po, To, key_bias=False):
    """Reverse sweep through (o, o-dot) = tangent(...): Po, To are the adjoints of o and
    o-dot.  Returns the adjoints of (q, k, v) and of (qd, kd, vd); with key_bias, also
    those of the key weights lu and of their tangents rho, each [n]."""
    c = np.sqrt(q.shape[1])
    p = weights(q, k, lu)
    zd = (qd @ k.T + q @ kd.T) / c + rho[None, :]
    zm = (p * zd).sum(1, keepdims=True)
    pd = p * (zd - zm)
    # o = p v, o-dot = pd v + p vd
    vb = p.T @ Po + pd.T @ To
    vdb = p.T @ To
    pb = Po @ v.T + To @ vd.T
    pdb = To @ v.T
    # pd = p * zd - p <p, zd>
    zdb = p * (pdb - (p * pdb).sum(1, keepdims=True))
    pb = pb + pdb * (zd - zm) - zd * (pdb * p).sum(1, keepdims=True)
    # p = softmax(z)
    zb = p * (pb - (p * pb).sum(1, keepdims=True))
    qb = (zb @ k + zdb @ kd) / c
    kb = (zb.T @ q + zdb.T @ qd) / c
    qdb = zdb @ k / c
    kdb = zdb.T @ q / c
    if key_bias:
        # z = q k^T / c + lu (per key), zd = (...) / c + rho (per key)
        return (qb, kb, vb), (qdb, kdb, vdb), (zb.sum(0), zdb.sum(0))
    return (qb, kb, vb), (qdb, kdb, vdb)
