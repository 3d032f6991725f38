"""Radial basis, envelope, SiLU family and Legendre polynomials (oracle).

Paper Sec. "MatRIS": pairwise distances are embedded as initial edge
features by the embedding module.  The paper prints no basis; the reading
used is the spherical-Bessel (DimeNet-style) radial basis

    B_n(r) = sqrt(2 / r_c) * sin(n pi r / r_c) / r * u(r / r_c),   n = 1..Nb

with the polynomial envelope of exponent p = 6

    u(x) = 1 - 28 x^6 + 48 x^7 - 21 x^8   (x < 1),   0 otherwise,

which has u(1) = u'(1) = u''(1) = 0, so B and its first two derivatives
vanish at the cutoff and the energy is twice differentiable there.  Without
the envelope the functions are orthonormal on [0, r_c] with weight r^2.

Derivatives are the closed forms of the product rule; everything is float64.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
from scipy.special import expit

_POOL = None


def _threads():
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:
        return os.cpu_count() or 1


def _rowwise(fn, a, n_out):
    """Apply an elementwise fn to row chunks of a on host threads (same values)."""
    global _POOL
    nt = _threads()
    if a.ndim < 1 or a.size < (1 << 20) or nt == 1 or a.shape[0] < nt:
        return fn(a)
    if _POOL is None:
        _POOL = ThreadPoolExecutor(nt)
    outs = [np.empty_like(a) for _ in range(n_out)]
    bounds = np.linspace(0, a.shape[0], nt + 1).astype(int)

    def work(c):
        res = fn(a[bounds[c]:bounds[c + 1]])
        for o, r in zip(outs, res):
            o[bounds[c]:bounds[c + 1]] = r
    list(_POOL.map(work, range(nt)))
    return tuple(outs)


def envelope(x):
    """u(x), du/dx, d2u/dx2 for the p = 6 polynomial envelope."""
    x = np.asarray(x, np.float64)
    inside = x < 1.0
    x5 = x ** 5
    u = np.where(inside, 1.0 - 28.0 * x ** 6 + 48.0 * x ** 7 - 21.0 * x ** 8, 0.0)
    du = np.where(inside, -168.0 * x5 + 336.0 * x5 * x - 168.0 * x5 * x * x, 0.0)
    d2u = np.where(inside, -840.0 * x ** 4 + 2016.0 * x5 - 1176.0 * x5 * x, 0.0)
    return u, du, d2u


def bessel_basis(r, r_cut, n_rbf):
    """B, dB/dr, d2B/dr2 at distances r [M] -> three [M, n_rbf] float64 arrays."""
    r = np.asarray(r, np.float64)[:, None]
    k = np.arange(1, n_rbf + 1, dtype=np.float64)[None, :] * np.pi / r_cut
    kr = k * r
    sn, cs = np.sin(kr), np.cos(kr)
    s = sn / r                                   # sin(kr)/r
    ds = (kr * cs - sn) / (r * r)                # d/dr
    d2s = -k * k * s - 2.0 * ds / r              # d2/dr2
    u, du, d2u = envelope(r / r_cut)
    ur, urr = du / r_cut, d2u / (r_cut * r_cut)
    c = np.sqrt(2.0 / r_cut)
    B = c * s * u
    dB = c * (ds * u + s * ur)
    d2B = c * (d2s * u + 2.0 * ds * ur + s * urr)
    return B, dB, d2B


def silu(a):
    """SiLU(a) = a * sigmoid(a)."""
    a = np.asarray(a, np.float64)
    return a * expit(a)


def silu_d1(a):
    """SiLU'(a) = s + a s (1 - s), s = sigmoid(a)."""
    a = np.asarray(a, np.float64)
    s = expit(a)
    return s + a * s * (1.0 - s)


def silu_d2(a):
    """SiLU''(a) = s (1 - s) (2 + a (1 - 2 s))."""
    a = np.asarray(a, np.float64)
    s = expit(a)
    return s * (1.0 - s) * (2.0 + a * (1.0 - 2.0 * s))


def _silu_family(a):
    s = expit(a)
    s1 = s * (1.0 - s)
    return a * s, s + a * s1, s1 * (2.0 + a * (1.0 - 2.0 * s))


def silu_family(a):
    """(SiLU, SiLU', SiLU'') of a from a single sigmoid evaluation."""
    return _rowwise(_silu_family, np.asarray(a, np.float64), 3)


def legendre2(x, n_l):
    """P_l(x), P_l'(x) and P_l''(x) for l = 0..n_l-1 -> [M, n_l] each: the Bonnet
    recurrence and its derivatives, (d/dx) P_{l+1} = (l+1) P_l + x P_l' and
    (d2/dx2) P_{l+1} = (l+2) P_l' + x P_l''."""
    P, dP = legendre(x, n_l)
    x = np.asarray(x, np.float64)
    d2P = np.zeros(x.shape + (n_l,))
    for l in range(1, n_l - 1):
        d2P[..., l + 1] = (l + 2) * dP[..., l] + x * d2P[..., l]
    return P, dP, d2P


def legendre(x, n_l):
    """P_l(x) and P_l'(x) for l = 0..n_l-1 (Bonnet recurrence) -> [M, n_l] each."""
    x = np.asarray(x, np.float64)
    P = np.zeros(x.shape + (n_l,))
    dP = np.zeros(x.shape + (n_l,))
    P[..., 0] = 1.0
    if n_l > 1:
        P[..., 1] = x
        dP[..., 1] = 1.0
    for l in range(1, n_l - 1):
        P[..., l + 1] = ((2 * l + 1) * x * P[..., l] - l * P[..., l - 1]) / (l + 1)
        # (d/dx) P_{l+1} = (l+1) P_l + x P_l'
        dP[..., l + 1] = (l + 1) * P[..., l] + x * dP[..., l]
    return P, dP
