"""janus_grouped_gemm_noalloc (the grouped GEMM with its tile table in the
library's fixed scratch, for callers that cannot allocate) through the C ABI
against janus_grouped_gemm on the same inputs: bitwise equal (the same
kernels over the same tiles) and within the float64 bound of the grouped
GEMM tests, on two calls in a row, the second smaller than the first (the
scratch keeps the first call's table); sizes beyond the scratch are refused
before any launch."""
import numpy as np
import pytest

from helpers import banner

pytestmark = pytest.mark.gpu


def _case(seed, sizes, K, N, trans_b):
    import torch
    rng = np.random.default_rng(seed)
    off = np.zeros(len(sizes) + 1, np.int32)
    off[1:] = np.cumsum(sizes)
    M, G = int(off[-1]), len(sizes)
    A = rng.standard_normal((M, K)).astype(np.float32)
    B = rng.standard_normal((G, N, K) if trans_b else (G, K, N)).astype(np.float32)
    return off, A, B, (torch.from_numpy(off).cuda(), torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda())


def _ref(off, A, B, trans_b):
    out = np.zeros((A.shape[0], B.shape[1] if trans_b else B.shape[2]))
    for g in range(len(off) - 1):
        a, b = off[g], off[g + 1]
        Bg = B[g].astype(np.float64)
        out[a:b] = A[a:b].astype(np.float64) @ (Bg.T if trans_b else Bg)
    return out


def test_noalloc_matches_grouped_gemm_on_two_calls():
    import torch
    from paper_2604_15821_amd import janus
    from paper_2604_15821_amd.synth import WORKLOADS
    ctx = janus.Context(WORKLOADS["tiny"].model)
    try:
        calls = [(1, [700, 0, 1300, 129, 5000, 1], 512, 256, 1),    # 62 tiles
                 (2, [3, 200, 0], 64, 128, 0)]                      # 4 tiles, smaller than the first
        for seed, sizes, K, N, tb in calls:
            banner("noalloc grouped_gemm", sizes, K, N, tb)
            off, A, B, (toff, tA, tB) = _case(seed, sizes, K, N, tb)
            M = A.shape[0]
            got = torch.full((M, N), float("nan"), device="cuda:0")
            janus.grouped_gemm_noalloc(tA, tB, toff, K, N, tb, out=got)
            want = torch.full((M, N), float("nan"), device="cuda:0")
            ctx.grouped_gemm(tA, tB, toff, K, N, tb, out=want)
            torch.cuda.synchronize()
            g, w = got.cpu().numpy(), want.cpu().numpy()
            assert np.isfinite(g).all()
            assert np.array_equal(g, w)
            ref = _ref(off, A, B, tb)
            err = np.abs(g - ref).max() / np.abs(ref).max()
            assert err < 2e-6 * np.sqrt(K), err
    finally:
        ctx.close()


def test_noalloc_refuses_sizes_beyond_the_scratch():
    """ceil(M / 128) + groups above 262128 tiles: refused before anything is launched."""
    import torch
    from paper_2604_15821_amd import janus
    A = torch.zeros(1, 16, device="cuda:0")
    B = torch.zeros(1, 16, 64, device="cuda:0")
    off = torch.zeros(2, dtype=torch.int32, device="cuda:0")
    C = torch.zeros(1, 64, device="cuda:0")
    lib = janus._lib()
    p = lambda t: janus._ptr(t)
    rc = lib.janus_grouped_gemm_noalloc(p(A), p(B), p(C), p(off), 1, 262127 * 128 + 1, 16, 64, 0, janus._stream())
    assert rc == janus.JANUS_ENOMEM
    torch.cuda.synchronize()
