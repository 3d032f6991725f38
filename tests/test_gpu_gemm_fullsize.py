"""Grouped GEMMs at the full-size expert shape (d = 512, h = 2048, 64 experts)
and length (over a million slot rows, the row count of one chunk of the
32,768-atom shard batch), through the C ABI, against float64.

Every entry of a product is one dot product, so sampled entries have an
exact float64 reference of their own; the column and row sums of each
weight-gradient block are one more contraction each (sum over p of G_g[p, q]
= sum over rows of (sum_p A[r, p]) B[r, q]), computed in float64 over every
row.  The rows are grouped like the irregular batch's routing: one
Zipf-heavy expert, a few empty ones, the rest log-uniform, with groups of
1, 127, 128, 2047, 2048 and 2049 rows at the tile and chunk boundaries.
Inputs are standard normal from a seeded device generator."""
import numpy as np
import pytest

from helpers import banner, rel_l2

pytestmark = pytest.mark.gpu

D, H, GROUPS = 512, 2048, 64
M_ROWS = 1_200_000
EMPTY = (5, 17, 40)
HEAVY = 23
EDGE_SIZES = {2: 1, 3: 127, 4: 128, 7: 2047, 8: 2048, 9: 2049}


def _row_offsets(seed):
    rng = np.random.default_rng(seed)
    w = np.exp(rng.uniform(0.0, np.log(50.0), GROUPS))
    w[list(EMPTY) + [HEAVY] + list(EDGE_SIZES)] = 0.0
    sizes = np.floor(w / w.sum() * (0.6 * M_ROWS)).astype(np.int64)
    for g, n in EDGE_SIZES.items():
        sizes[g] = n
    sizes[HEAVY] = M_ROWS - sizes.sum()
    assert sizes[HEAVY] > 0.35 * M_ROWS and all(sizes[g] == 0 for g in EMPTY)
    off = np.zeros(GROUPS + 1, np.int32)
    off[1:] = np.cumsum(sizes)
    return off


def _randn(shape, seed):
    import torch
    g = torch.Generator(device="cuda:0")
    g.manual_seed(seed)
    return torch.randn(shape, generator=g, device="cuda:0", dtype=torch.float32)


@pytest.fixture(scope="module")
def ctx():
    from paper_2604_15821_amd import janus
    from paper_2604_15821_amd.synth import WORKLOADS
    c = janus.Context(WORKLOADS["tiny"].model)
    yield c
    c.close()


def _sample_rows(off, n, seed):
    """Rows at the ends of every group and of its first tiles, plus random rows."""
    rng = np.random.default_rng(seed)
    rows = []
    for g in range(GROUPS):
        a, b = int(off[g]), int(off[g + 1])
        if b > a:
            rows += [r for r in (a, a + 127, a + 128, b - 1) if a <= r < b]
    rows += list(rng.integers(0, int(off[-1]), n - len(rows)))
    return np.unique(np.asarray(rows, np.int64))


@pytest.mark.parametrize("K,N,trans_b", [(D, H, 0), (H, D, 1), (H, D, 0), (D, H, 1)])
def test_grouped_gemm_full_size_sampled_rows(ctx, K, N, trans_b):
    import torch
    banner("grouped_gemm full size", M_ROWS, "rows", K, N, "NT" if trans_b else "NN")
    off = _row_offsets(1)
    A = _randn((M_ROWS, K), 11 + K)
    B = _randn((GROUPS, N, K) if trans_b else (GROUPS, K, N), 12 + N) * (1.0 / np.sqrt(K))
    C = torch.full((M_ROWS, N), float("nan"), device="cuda:0")
    ctx.grouped_gemm(A, B, torch.from_numpy(off).cuda(), K, N, trans_b, out=C)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(C).all())
    rows = _sample_rows(off, 4096, 3)
    idx = torch.from_numpy(rows).cuda()
    a = A[idx].cpu().numpy().astype(np.float64)
    got = C[idx].cpu().numpy()
    grp = np.searchsorted(off, rows, side="right") - 1
    Bh = B.cpu().numpy()
    ref = np.empty_like(got, dtype=np.float64)
    for g in np.unique(grp):
        sel = grp == g
        Bg = Bh[g].astype(np.float64)
        ref[sel] = a[sel] @ (Bg.T if trans_b else Bg)
    err = np.abs(got - ref).max() / np.abs(ref).max()
    print(f"  {len(rows)} rows, max error / max |C| = {err:.2e}", flush=True)
    assert err < 2e-6 * np.sqrt(K), err


def test_grouped_wgrad_full_size(ctx):
    """G_g = A_g^T B_g with P = d, Q = h over 1.2 M rows: 2048-row chunks (the length the
    expert weight gradients of the full-size workloads use), 4096 sampled entries and
    every column and row sum against float64, empty experts exactly zero."""
    import torch
    from paper_2604_15821_amd import janus
    P, Q = D, H
    kc = janus.wgrad_chunk_rows(M_ROWS, P, Q)
    assert kc == 2048
    banner("grouped_wgrad full size", M_ROWS, "rows", P, Q, "chunk", kc)
    off = _row_offsets(2)
    A = _randn((M_ROWS, P), 21)
    B = _randn((M_ROWS, Q), 22)
    G = torch.full((GROUPS, P, Q), float("nan"), device="cuda:0")
    ctx.grouped_wgrad(A, B, torch.from_numpy(off).cuda(), out=G)
    torch.cuda.synchronize()
    got = G.cpu().numpy()
    assert np.isfinite(got).all()
    for g in EMPTY:
        assert (got[g] == 0).all(), g
    Ah = A.cpu().numpy()
    Bh = B.cpu().numpy()
    del A, B
    torch.cuda.empty_cache()

    rng = np.random.default_rng(4)
    nonempty = [g for g in range(GROUPS) if off[g + 1] > off[g]]
    worst_entry, col_errs, row_errs = 0.0, [], []
    got_s, ref_s = [], []
    step = 65536
    for g in nonempty:
        a0, a1 = int(off[g]), int(off[g + 1])
        ps = np.sort(rng.choice(P, 9, replace=False))
        qs = np.sort(rng.choice(Q, 8, replace=False))
        ref = np.zeros((9, 8))
        scale = np.zeros((9, 8))
        colsum = np.zeros(Q)      # sum over p of G_g[p, q]
        rowsum = np.zeros(P)      # sum over q of G_g[p, q]
        for r0 in range(a0, a1, step):
            r1 = min(r0 + step, a1)
            a = Ah[r0:r1].astype(np.float64)
            b = Bh[r0:r1].astype(np.float64)
            ref += a[:, ps].T @ b[:, qs]
            scale += (a[:, ps] ** 2).T @ (b[:, qs] ** 2)
            colsum += a.sum(1) @ b
            rowsum += a.T @ b.sum(1)
        e = np.abs(got[g][np.ix_(ps, qs)] - ref) / np.sqrt(scale)
        worst_entry = max(worst_entry, float(e.max()))
        got_s.append(got[g][np.ix_(ps, qs)].ravel())
        ref_s.append(ref.ravel())
        col_errs.append(rel_l2(got[g].astype(np.float64).sum(0), colsum))
        row_errs.append(rel_l2(got[g].astype(np.float64).sum(1), rowsum))
    samp = rel_l2(np.concatenate(got_s), np.concatenate(ref_s))
    n_entries = sum(x.size for x in got_s)
    print(f"  {len(nonempty)} experts, {n_entries} sampled entries: worst |error| / sqrt(sum a^2 b^2) "
          f"{worst_entry:.2e}, rel L2 {samp:.2e}; column sums {max(col_errs):.2e}, row sums {max(row_errs):.2e}",
          flush=True)
    assert n_entries >= 4096
    assert worst_entry < 1e-4
    assert samp < 2e-5
    assert max(col_errs) < 2e-5 and max(row_errs) < 2e-5
