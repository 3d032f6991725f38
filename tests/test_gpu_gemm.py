"""Grouped fp32-MFMA GEMMs through the C ABI against float64 matrix products
(the plain definition of each grouped product)."""
import numpy as np
import pytest

from helpers import banner, rel_l2

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    import torch
    from paper_2604_15821_amd import janus
    from paper_2604_15821_amd.synth import WORKLOADS
    c = janus.Context(WORKLOADS["tiny"].model)
    yield c
    c.close()


def _groups(rng, sizes):
    off = np.zeros(len(sizes) + 1, np.int32)
    off[1:] = np.cumsum(sizes)
    return off


CASES = [
    # (group sizes, K, N)
    ([0, 1, 127, 128, 129, 300, 0, 5], 64, 128),
    ([513, 0, 77], 128, 512),
    ([1000, 260], 512, 128),
    ([3], 16, 64),
    ([0, 0], 64, 64),
    # a last column tile with 64 of its 128 columns (and rows of 130 and 7)
    ([130, 0, 7], 32, 192),
    ([64, 200], 96, 320),
]


@pytest.mark.parametrize("sizes,K,N", CASES)
@pytest.mark.parametrize("trans_b", [0, 1])
def test_grouped_gemm_matches_float64(ctx, sizes, K, N, trans_b):
    import torch
    banner("grouped_gemm", sizes, K, N, trans_b)
    rng = np.random.default_rng(len(sizes) * 100 + K + N + trans_b)
    off = _groups(rng, sizes)
    M = int(off[-1])
    G = len(sizes)
    A = rng.standard_normal((M, K)).astype(np.float32)
    B = rng.standard_normal((G, N, K) if trans_b else (G, K, N)).astype(np.float32)
    dev = "cuda:0"
    tA = torch.from_numpy(A).to(dev)
    tB = torch.from_numpy(B).to(dev)
    toff = torch.from_numpy(off).to(dev)
    out = torch.full((M, N), float("nan"), device=dev)
    ctx.grouped_gemm(tA, tB, toff, K, N, trans_b, out=out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    ref = np.zeros((M, N))
    for g in range(G):
        a, b = off[g], off[g + 1]
        Bg = B[g].astype(np.float64)
        ref[a:b] = A[a:b].astype(np.float64) @ (Bg.T if trans_b else Bg)
    assert np.isfinite(got).all()
    if M:
        err = np.abs(got - ref).max() / max(np.abs(ref).max(), 1e-30)
        assert err < 2e-6 * np.sqrt(K), err


WG_CASES = [
    ([0, 1, 2047, 2048, 2049, 5000, 0], 64, 128),
    ([7000, 0, 300], 128, 512),
    ([4097], 16, 128),
    ([513, 20], 512, 128),
    ([0, 0, 0], 8, 64),
    # partial column tiles on both sides, chunks ending inside and on a 16-row stage
    ([300, 45, 0, 16], 192, 64),
    ([1000], 48, 320),
]


@pytest.mark.parametrize("sizes,P,Q", WG_CASES)
def test_grouped_wgrad_matches_float64(ctx, sizes, P, Q):
    import torch
    banner("grouped_wgrad", sizes, P, Q)
    rng = np.random.default_rng(P * 7 + Q + len(sizes))
    off = _groups(rng, sizes)
    M = int(off[-1])
    G = len(sizes)
    A = rng.standard_normal((M, P)).astype(np.float32)
    B = rng.standard_normal((M, Q)).astype(np.float32)
    dev = "cuda:0"
    out = torch.full((G, P, Q), float("nan"), device=dev)
    ctx.grouped_wgrad(torch.from_numpy(A).to(dev), torch.from_numpy(B).to(dev), torch.from_numpy(off).to(dev),
                      out=out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    for g in range(G):
        a, b = off[g], off[g + 1]
        ref = A[a:b].astype(np.float64).T @ B[a:b].astype(np.float64)
        if b == a:
            assert (got[g] == 0).all()
        else:
            assert rel_l2(got[g], ref) < 1e-5, (g, rel_l2(got[g], ref))


def test_wgrad_is_deterministic(ctx):
    import torch
    banner("wgrad determinism")
    rng = np.random.default_rng(5)
    off = _groups(rng, [9000, 3000])
    A = torch.from_numpy(rng.standard_normal((12000, 128)).astype(np.float32)).cuda()
    B = torch.from_numpy(rng.standard_normal((12000, 256)).astype(np.float32)).cuda()
    o = torch.from_numpy(off).cuda()
    r1 = ctx.grouped_wgrad(A, B, o).cpu().numpy()
    r2 = ctx.grouped_wgrad(A, B, o).cpu().numpy()
    assert (r1 == r2).all()
