"""Writes threebody_full.npz: the float64 oracle's training step on the whole
64-structure three-body batch (4,096 atoms, about 846 k bond triplets), which
takes several minutes on the host, too long to repeat inside a GPU test.

Stored: the loss; E [S] and the per-structure norm of the per-atom energies
(the guard of the energy tolerance); F [N, 3]; and for every weight-gradient
tensor its L2 norm, a count sketch of 1024 buckets (seeded buckets and signs,
see tests/helpers.py; tensors of at most 4096 entries are stored whole) and
256 seeded sampled entries.  Calls only the oracle and the input generator.

    python tests/golden/make_threebody_full.py
"""
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.dirname(HERE))

from helpers import count_sketch, sketch_keys  # noqa: E402

SEED = 2026
K = 1024
WHOLE = 4096
SAMPLES = 256


def main():
    from oracle.model import Params, forward_energy, training_step
    from paper_2604_15821_amd.synth import make_batch
    b = make_batch("threebody")
    loss, E, F, grad, aux = training_step(b, return_aux=True)
    _, cache = forward_energy(b.species, aux["graph"], Params.from_weights(b.weights, b.model), aux["routing"])
    eps = cache["eps"]
    eps_norm = np.array([np.linalg.norm(eps[b.offsets[s]:b.offsets[s + 1]]) for s in range(b.n_struct)])
    out = {"loss": np.float64(loss), "E": E, "eps_norm": eps_norm, "F": F,
           "n_edges": np.int64(aux["graph"].ei.size), "n_triplets": np.int64(aux["graph"].tri.te.size)}
    names = sorted(grad)
    out["names"] = np.array(names)
    for q, name in enumerate(names):
        g = np.asarray(grad[name], np.float64).ravel()
        out[f"norm/{name}"] = np.float64(np.linalg.norm(g))
        if g.size <= WHOLE:
            out[f"whole/{name}"] = g
        else:
            out[f"sketch/{name}"] = count_sketch(g, sketch_keys(SEED, q, g.size, K), K)
        idx = np.random.default_rng([SEED, q, 1]).integers(0, g.size, min(SAMPLES, g.size))
        out[f"samples/{name}"] = g[idx]
    path = os.path.join(HERE, "threebody_full.npz")
    np.savez_compressed(path, **out)
    print(path, os.path.getsize(path), "bytes; loss", loss)


if __name__ == "__main__":
    main()
