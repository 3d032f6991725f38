"""Shared helpers of the GPU parity tests (comparisons and case banners)."""
import sys

import numpy as np


def banner(*parts):
    """Name the case on stdout before a GPU step, so a failed run says what ran."""
    print("[case]", *parts, flush=True)
    sys.stdout.flush()


def rel_l2(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    if den == 0.0:
        return float(np.linalg.norm(got))
    return float(np.linalg.norm(got - ref) / den)


def energy_error(E_gpu, E_ref, eps_ref, offsets):
    """max_s |dE_s| / max(|E_s|, ||eps_{i in s}||_2): relative energy error with a
    guard against cancellation inside a structure."""
    worst = 0.0
    for s in range(len(E_ref)):
        a, b = int(offsets[s]), int(offsets[s + 1])
        scale = max(abs(float(E_ref[s])), float(np.linalg.norm(eps_ref[a:b])))
        worst = max(worst, abs(float(E_gpu[s]) - float(E_ref[s])) / scale)
    return worst


# Tolerances of the floating-point outputs (energy 1e-5 relative, forces and
# every weight gradient 1e-3 relative L2); integer outputs are compared exactly.
TOL_E = 1e-5
TOL_LOSS = 1e-5
TOL_F = 1e-3
TOL_W = 1e-3


def sketch_keys(seed, index, n, K):
    """Bucket and sign of every entry for the count sketch of tensor number `index`
    (seeded, so the expected sketch can be stored and the measured one recomputed)."""
    rng = np.random.default_rng([seed, index])
    return rng.integers(0, K, n), rng.integers(0, 2, n) * 2.0 - 1.0


def count_sketch(x, keys, K):
    """Linear sketch of a tensor: bucket k holds the sum of s_i x_i over the entries i
    hashed to k.  For any vector v, |sketch(v)|^2 is an unbiased estimate of |v|^2 with
    relative standard deviation at most sqrt(2 / K), so |sketch(a) - sketch(b)| estimates
    |a - b| (the relative L2 error of a stored tensor) without storing the tensor."""
    h, s = keys
    return np.bincount(h, weights=s * np.asarray(x, np.float64).ravel(), minlength=K)
