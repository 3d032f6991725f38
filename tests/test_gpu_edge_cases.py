"""Degenerate inputs of the training step against the oracle: structures
whose atoms have no neighbours (isolated atoms, and a batch without a single
edge), three-body batches without triplets (dimers) or with very few
(a triangle), and the three-body step split into several chunks.

Isolated structures place their atoms on a cubic grid of 10 A spacing in a
box whose images are at least 10 A away, so no pair is within any cutoff
used here; dimers and triangles use 3 A bonds in a 30 A box."""
import dataclasses

import numpy as np
import pytest

from helpers import TOL_E, TOL_F, TOL_LOSS, TOL_W, banner, energy_error, rel_l2

pytestmark = pytest.mark.gpu


def _replace_structs(b, structs, make):
    """Batch b with the positions and cell of the listed structures replaced by make(n_atoms)."""
    pos, cell = b.pos.copy(), b.cell.copy()
    for s in structs:
        a0, a1 = int(b.offsets[s]), int(b.offsets[s + 1])
        p, L = make(a1 - a0)
        pos[a0:a1] = p
        cell[s] = np.diag([L, L, L]).astype(np.float32)
    return dataclasses.replace(b, pos=pos.astype(np.float32), cell=cell)


def _grid(n, spacing=10.0):
    m = int(np.ceil(n ** (1.0 / 3.0)))
    idx = np.array([(x, y, z) for x in range(m) for y in range(m) for z in range(m)][:n], np.float64)
    return (idx * spacing + 1.0).astype(np.float32), np.float32(m * spacing + spacing)


def _gpu(b, limit=None, reps=1):
    import torch
    from paper_2604_15821_amd import janus
    d = janus.upload(b)
    ctx = janus.Context(b.model)
    if limit is not None:
        ctx.set_workspace_limit(limit)
    try:
        nl = ctx.build_edges(d["pos"], d["cell"], d["offsets"])
        outs = []
        for _ in range(reps):
            loss, E, F, dW = ctx.step(d["pos"], d["cell"], d["species"], d["offsets"], nl, d["W"], d["E_ref"],
                                      d["F_ref"])
            torch.cuda.synchronize()
            outs.append({"loss": float(loss.cpu()[0]), "E": E.cpu().numpy(), "F": F.cpu().numpy(),
                         "dW": dW.cpu().numpy()})
        info = {"edges": nl.n_edges, "chunks": ctx.last_chunks(), "triplets": ctx.last_triplets()}
    finally:
        ctx.close()
    return outs, info


def _check_against_oracle(b, out):
    from oracle.model import Params, forward_energy, training_step
    from paper_2604_15821_amd import janus
    loss, E, F, grad, aux = training_step(b, return_aux=True)
    _, cache = forward_energy(b.species, aux["graph"], Params.from_weights(b.weights, b.model), aux["routing"])
    assert energy_error(out["E"], E, cache["eps"], b.offsets) <= TOL_E
    assert abs(out["loss"] - loss) <= TOL_LOSS * abs(loss)
    if np.linalg.norm(F) > 0:
        assert rel_l2(out["F"], F) <= TOL_F
    else:
        assert not out["F"].any()
    got = janus.unpack(out["dW"], b.model)
    for name, ref in grad.items():
        if name.endswith("beta"):
            continue
        if not ref.any():
            assert not got[name].any(), name       # exact zeros where the oracle has none
        else:
            assert rel_l2(got[name], ref) <= TOL_W, (name, rel_l2(got[name], ref))
    return aux


def test_structure_with_isolated_atoms():
    from paper_2604_15821_amd.synth import make_batch, subset
    b = _replace_structs(subset(make_batch("tiny"), range(4)), [1], _grid)
    banner("edge cases: tiny-4 with structure 1 isolated")
    (out,), info = _gpu(b)
    a0, a1 = b.offsets[1], b.offsets[2]
    assert not out["F"][a0:a1].any()
    aux = _check_against_oracle(b, out)
    g = aux["graph"]
    assert info["edges"] == g.ei.size and not ((g.ei >= a0) & (g.ei < a1)).any()


def test_batch_without_edges():
    from paper_2604_15821_amd.synth import make_batch, subset
    b = _replace_structs(subset(make_batch("tiny"), range(2)), [0, 1], _grid)
    banner("edge cases: tiny-2, no edges at all")
    (out,), info = _gpu(b)
    assert info["edges"] == 0
    assert not out["F"].any()
    _check_against_oracle(b, out)


def _dimer(n):
    p = np.zeros((n, 3), np.float32)
    p[1, 0] = 3.0
    return p + 1.0, np.float32(30.0)


def _triangle(n):
    p = np.zeros((n, 3), np.float32)
    p[1] = (3.0, 0.0, 0.0)
    p[2] = (1.5, 1.5 * np.sqrt(3.0), 0.0)
    return p + 1.0, np.float32(30.0)


def _small_molecules(shapes):
    """Three-body batch of len(shapes) molecules of 2 or 3 atoms (species and weights from the workload)."""
    from paper_2604_15821_amd.synth import make_batch
    base = make_batch("threebody")
    sizes = [2 if s == "dimer" else 3 for s in shapes]
    off = np.zeros(len(sizes) + 1, np.int32)
    off[1:] = np.cumsum(sizes)
    n = int(off[-1])
    b = dataclasses.replace(base, pos=np.zeros((n, 3), np.float32), cell=base.cell[:len(sizes)].copy(),
                            species=base.species[:n].copy(), offsets=off, E_ref=base.E_ref[:len(sizes)].copy(),
                            F_ref=base.F_ref[:n].copy())
    for s, kind in enumerate(shapes):
        b = _replace_structs(b, [s], _dimer if kind == "dimer" else _triangle)
    return b


def test_three_body_batch_without_triplets():
    b = _small_molecules(["dimer", "dimer", "dimer"])
    banner("edge cases: three-body dimers")
    (out,), info = _gpu(b)
    assert info["edges"] == 6 and info["triplets"] == 0
    _check_against_oracle(b, out)


def test_three_body_triangle_among_dimers():
    b = _small_molecules(["dimer", "triangle", "dimer"])
    banner("edge cases: three-body triangle")
    (out,), info = _gpu(b)
    assert info["edges"] == 10 and info["triplets"] == 6
    aux = _check_against_oracle(b, out)
    assert aux["graph"].tri.te.size == 6


def test_three_body_chunked_matches_single_pass_and_oracle():
    from paper_2604_15821_amd.synth import make_batch, subset
    b = subset(make_batch("threebody"), range(4))
    banner("edge cases: threebody-4 in chunks")
    from paper_2604_15821_amd import janus
    (o1,), i1 = _gpu(b)
    # the smallest of these caps that fits one structure splits the batch
    for limit in (2e8, 3e8, 4.5e8, 7e8):
        try:
            (o2,), i2 = _gpu(b, limit=int(limit))
            break
        except janus.JanusError:
            continue
    print("cap", limit, "chunks", i1["chunks"], i2["chunks"], "triplets", i2["triplets"], flush=True)
    assert i1["chunks"] == 1 and i2["chunks"] >= 2 and i1["triplets"] == i2["triplets"] > 0
    assert (o1["E"] == o2["E"]).all() and (o1["F"] == o2["F"]).all()
    assert abs(o1["loss"] - o2["loss"]) <= 1e-6 * abs(o1["loss"])
    assert rel_l2(o2["dW"], o1["dW"]) <= 1e-6
    _check_against_oracle(b, o2)


@pytest.mark.parametrize("what", ["species", "edge_index", "reverse_map", "offsets"])
def test_step_rejects_invalid_inputs(what):
    """Invalid species, neighbour lists or offsets are refused before any compute
    (the validation kernels read only in-range indices)."""
    import torch
    from paper_2604_15821_amd import janus
    from paper_2604_15821_amd.synth import make_batch, subset
    b = subset(make_batch("tiny"), range(2))
    banner("edge cases: invalid", what)
    d = janus.upload(b)
    ctx = janus.Context(b.model)
    try:
        nl = ctx.build_edges(d["pos"], d["cell"], d["offsets"])
        offsets = d["offsets"]
        if what == "species":
            d["species"][3] = b.model.n_species
        elif what == "edge_index":
            nl.ej[0] = b.n_atoms + 5
        elif what == "reverse_map":
            nl.rev[0] = nl.rev[1]
        else:
            offsets = offsets.clone()
            offsets[-1] = b.n_atoms - 1
        torch.cuda.synchronize()
        with pytest.raises(janus.JanusError) as ex:
            ctx.step(d["pos"], d["cell"], d["species"], offsets, nl, d["W"], d["E_ref"], d["F_ref"])
        assert ex.value.code == janus.JANUS_EINVAL
    finally:
        ctx.close()
