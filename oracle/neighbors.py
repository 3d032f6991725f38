"""Periodic neighbour list, reverse-edge map and bond triplets (oracle).

Paper Sec. "MatRIS": a structure G(Z, X, L) is periodically repeated and
turned into an atom graph with bond edges and bond-pair angles by the graph
generation module.  The paper gives no inclusion rule; the reading used here
(and by the HIP path, which must match it bit for bit) is:

* An edge e = (i, j, n) joins atom i to the image of atom j shifted by the
  integer lattice vector n, with i, j in the same structure and
  (i, n) != (j, 0).
* The displacement is evaluated in float32 with a fixed operation order and
  no fused multiply-add:
      shift_k = (n_a * a_k + n_b * b_k) + n_c * c_k
      d_k     = (X_j,k - X_i,k) + shift_k
      r2      = (d_x * d_x + d_y * d_y) + d_z * d_z
  and the edge is kept iff r2 < float32(r_cut) * float32(r_cut).
* Images n_k range over [-m_k, m_k] with m_k = floor(r_cut * |b_k|) + 1,
  b_k the reciprocal vectors (for an orthorhombic cell, floor(r_cut/L_k)+1).
  This covers every hit when positions are wrapped into the cell.
* Edges are listed in lexicographic (i, j, n_a, n_b, n_c) order.

NumPy float32 ufuncs round each operation to float32 separately, so the
expressions above are evaluated exactly as written.
"""
from __future__ import annotations

import itertools

import numpy as np


def image_range(cell: np.ndarray, r_cut: float) -> tuple[int, int, int]:
    """Half-widths m_k of the image box for one cell (rows a, b, c)."""
    c64 = np.asarray(cell, np.float64)
    if np.count_nonzero(c64 - np.diag(np.diag(c64))) == 0:
        return tuple(int(np.floor(float(r_cut) / c64[k, k])) + 1 for k in range(3))
    recip = np.linalg.inv(c64).T
    return tuple(int(np.floor(float(r_cut) * np.linalg.norm(recip[k]))) + 1 for k in range(3))


def _images(m):
    rng = [range(-mk, mk + 1) for mk in m]
    return np.array(list(itertools.product(*rng)), dtype=np.int64)  # lexicographic


def neighbor_list(pos, cell, offsets, r_cut):
    """All edges of the batch under the pinned float32 test.

    pos [N,3], cell [S,3,3] (rows are lattice vectors), offsets [S+1].
    Returns (ei, ej, shift, rowptr): int32 [Ne], int32 [Ne], int8 [Ne,3],
    int32 [N+1] (CSR by centre atom i).
    """
    pos32 = np.asarray(pos, np.float32)
    cell32 = np.asarray(cell, np.float32)
    rc = np.float32(r_cut)
    rc2 = rc * rc
    N = pos32.shape[0]
    ei_l, ej_l, sh_l = [], [], []
    for s in range(cell32.shape[0]):
        a, b = int(offsets[s]), int(offsets[s + 1])
        n = b - a
        if n == 0:
            continue
        img = _images(image_range(cell32[s], r_cut))
        imf = img.astype(np.float32)
        L = cell32[s]
        # shift_k = (na*a_k + nb*b_k) + nc*c_k, each product and sum in float32
        shift = (imf[:, 0:1] * L[0][None, :] + imf[:, 1:2] * L[1][None, :]) + imf[:, 2:3] * L[2][None, :]
        shift = shift.astype(np.float32)
        p = pos32[a:b]
        zero = int(np.nonzero((img == 0).all(1))[0][0])
        # centres in blocks of rows (the [i, j, img] arrays of a large structure would not
        # fit in memory); blocks in order keep the canonical order
        blk = max(1, int(2e7 // (n * img.shape[0])))
        for i0 in range(0, n, blk):
            i1 = min(n, i0 + blk)
            diff = p[None, :, :] - p[i0:i1, None, :]                  # [i, j, 3] = X_j - X_i
            dvec = diff[:, :, None, :] + shift[None, None, :, :]      # [i, j, img, 3]
            dx, dy, dz = dvec[..., 0], dvec[..., 1], dvec[..., 2]
            r2 = (dx * dx + dy * dy) + dz * dz
            keep = r2 < rc2
            idx = np.arange(i0, i1)
            keep[idx - i0, idx, zero] = False
            ii, jj, kk = np.nonzero(keep)                              # C order = canonical order
            ei_l.append((ii + a + i0).astype(np.int32))
            ej_l.append((jj + a).astype(np.int32))
            sh_l.append(img[kk].astype(np.int8))
    if ei_l:
        ei = np.concatenate(ei_l)
        ej = np.concatenate(ej_l)
        sh = np.concatenate(sh_l).reshape(-1, 3)
    else:
        ei = np.zeros(0, np.int32); ej = np.zeros(0, np.int32); sh = np.zeros((0, 3), np.int8)
    rowptr = np.zeros(N + 1, np.int32)
    rowptr[1:] = np.cumsum(np.bincount(ei, minlength=N))
    return ei, ej, sh, rowptr


def _edge_key(i, j, sh, N):
    s = sh.astype(np.int64) + 16
    return ((i.astype(np.int64) * N + j.astype(np.int64)) * 32 + s[:, 0]) * 1024 + s[:, 1] * 32 + s[:, 2]


def reverse_map(ei, ej, shift, N):
    """rev[e] = index of the edge (j, i, -n); raises if the list is not symmetric."""
    key = _edge_key(ei, ej, shift, N)
    if key.size > 1 and not np.all(np.diff(key) > 0):
        raise ValueError("edge list is not in canonical order")
    rkey = _edge_key(ej, ei, -shift.astype(np.int64), N)
    rev = np.searchsorted(key, rkey)
    ok = (rev < key.size)
    ok[ok] &= key[rev[ok]] == rkey[ok]
    if not np.all(ok):
        raise ValueError("edge list is not symmetric")
    return rev.astype(np.int32)


def triplet_list(ei, ej, shift, pos, cell, offsets, rowptr, r_cut3):
    """Ordered bond pairs (e, e2) sharing the centre atom, both bonds short.

    Paper Sec. "MatRIS": angles a_ijk are formed by two bonds sharing an atom.
    Reading: a triplet is an ordered pair of distinct edges e = (i, j, n),
    e2 = (i, k, n') out of the same centre i whose pinned float32 r2 are both
    below float32(r_cut3)^2; listed in lexicographic (e, e2) order.
    Returns (te, te2) int32 [Nt] and trowptr int32 [Ne+1] (CSR by e).
    """
    pos32 = np.asarray(pos, np.float32)
    cell32 = np.asarray(cell, np.float32)
    Ne = ei.shape[0]
    N = pos32.shape[0]
    sid = np.zeros(N, np.int64)
    for s in range(cell32.shape[0]):
        sid[int(offsets[s]):int(offsets[s + 1])] = s
    L = cell32[sid[ei]]                                            # [Ne, 3, 3]
    imf = shift.astype(np.float32)
    sh = (imf[:, 0:1] * L[:, 0] + imf[:, 1:2] * L[:, 1]) + imf[:, 2:3] * L[:, 2]
    d = (pos32[ej] - pos32[ei]) + sh.astype(np.float32)
    r2 = (d[:, 0] * d[:, 0] + d[:, 1] * d[:, 1]) + d[:, 2] * d[:, 2]
    rc3 = np.float32(r_cut3)
    short = r2 < rc3 * rc3
    te_l, te2_l = [], []
    for i in range(N):
        lo, hi = int(rowptr[i]), int(rowptr[i + 1])
        es = np.arange(lo, hi)[short[lo:hi]]
        if es.size < 2:
            continue
        a = np.repeat(es, es.size)
        b = np.tile(es, es.size)
        m = a != b
        te_l.append(a[m]); te2_l.append(b[m])
    if te_l:
        te = np.concatenate(te_l).astype(np.int32); te2 = np.concatenate(te2_l).astype(np.int32)
    else:
        te = np.zeros(0, np.int32); te2 = np.zeros(0, np.int32)
    trowptr = np.zeros(Ne + 1, np.int32)
    trowptr[1:] = np.cumsum(np.bincount(te, minlength=Ne))
    return te, te2, trowptr
