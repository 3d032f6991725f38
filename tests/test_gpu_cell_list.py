"""Cell-list candidate search of the edge builder (janus_set_edge_builder)
against the oracle: the neighbour list is bit-exact in every mode (cell list
everywhere, all pairs everywhere, automatic) on the workload batches, on a
5,000-atom cell (where the automatic mode takes the cell list), on a batch
that mixes it with small structures and an empty one, on positions far
outside their cell, and on a dense cell whose centres keep more than the
512 neighbours the cell-list write pass sorts (written by the all-pairs
kernel)."""
import time

import numpy as np
import pytest

from helpers import banner

pytestmark = pytest.mark.gpu

AUTO, CELLS, PAIRS = 0, 1, 2


def _model(r_cut):
    import dataclasses
    from paper_2604_15821_amd.synth import WORKLOADS
    return dataclasses.replace(WORKLOADS["tiny"].model, r_cut=r_cut)


def _build(model, pos, cell, offsets, mode):
    import torch
    from paper_2604_15821_amd import janus
    ctx = janus.Context(model)
    try:
        ctx.set_edge_builder(mode)
        p = torch.from_numpy(np.ascontiguousarray(pos, np.float32)).cuda()
        c = torch.from_numpy(np.ascontiguousarray(cell, np.float32)).cuda()
        o = torch.from_numpy(np.ascontiguousarray(offsets, np.int32)).cuda()
        ctx.build_edges(p, c, o)                          # sizes the buffers
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        nl = ctx.build_edges(p, c, o)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        out = {k: getattr(nl, k).cpu().numpy() for k in ("ei", "ej", "shift", "rowptr", "rev")}
        out["n"] = nl.n_edges
        out["ms"] = dt * 1e3
    finally:
        ctx.close()
    return out


def _check(got, pos, cell, offsets, r_cut):
    from oracle.neighbors import neighbor_list, reverse_map
    ei, ej, sh, rp = neighbor_list(pos, cell, offsets, r_cut)
    assert got["n"] == ei.shape[0]
    assert (got["ei"] == ei).all() and (got["ej"] == ej).all()
    assert (got["shift"] == sh).all() and (got["rowptr"] == rp).all()
    assert (got["rev"] == reverse_map(ei, ej, sh, pos.shape[0])).all()
    return ei.shape[0]


@pytest.mark.parametrize("name,n", [("tiny", None), ("small", 6), ("shard", 2), ("irregular", 24)])
@pytest.mark.parametrize("mode", [CELLS, PAIRS, AUTO])
def test_workload_batches_every_mode(name, n, mode):
    from paper_2604_15821_amd.synth import make_batch, subset
    b = make_batch(name)
    if n is not None:
        b = subset(b, range(n))
    banner("cell list", name, n, "mode", mode)
    got = _build(b.model, b.pos, b.cell, b.offsets, mode)
    _check(got, b.pos, b.cell, b.offsets, b.model.r_cut)


def _large_cell(n=5000, L=40.0, seed=11):
    rng = np.random.default_rng(seed)
    return (rng.random((n, 3)) * L).astype(np.float32), np.diag([L] * 3).astype(np.float32)


def test_large_cell_automatic_mode_matches_oracle():
    pos, cell = _large_cell()
    offsets = np.array([0, pos.shape[0]], np.int32)
    banner("cell list large cell", pos.shape[0], "atoms")
    auto = _build(_model(6.0), pos, cell[None], offsets, AUTO)
    pairs = _build(_model(6.0), pos, cell[None], offsets, PAIRS)
    ne = _check(auto, pos, cell[None], offsets, 6.0)
    for k in ("ei", "ej", "shift", "rowptr", "rev"):
        assert (auto[k] == pairs[k]).all(), k
    print(f"  {ne} edges; build {auto['ms']:.2f} ms (cell list) against {pairs['ms']:.2f} ms (all pairs)",
          flush=True)


def test_mixed_batch_with_an_empty_structure():
    from paper_2604_15821_amd.synth import make_batch, subset
    small = subset(make_batch("tiny"), range(3))
    big, bcell = _large_cell(n=4096, L=36.0, seed=12)
    pos = np.concatenate([small.pos[: small.offsets[2]], big, small.pos[small.offsets[2]:]]).astype(np.float32)
    sizes = [small.offsets[1], small.offsets[2] - small.offsets[1], big.shape[0], 0,
             small.offsets[3] - small.offsets[2]]
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    cell = np.stack([small.cell[0], small.cell[1], bcell, small.cell[2], small.cell[2]]).astype(np.float32)
    r_cut = 4.0
    banner("cell list mixed batch", pos.shape[0], "atoms")
    for mode in (AUTO, CELLS, PAIRS):
        _check(_build(_model(r_cut), pos, cell, offsets, mode), pos, cell, offsets, r_cut)


def test_positions_outside_the_cell():
    """Unwrapped coordinates (atoms moved by whole and fractional box lengths): the list
    is defined by the test over the image range, and both searches reproduce it."""
    rng = np.random.default_rng(13)
    L = 9.0
    pos = (rng.random((300, 3)) * L + rng.integers(-3, 4, (300, 3)) * L * 0.5).astype(np.float32)
    cell = np.diag([L] * 3).astype(np.float32)[None]
    offsets = np.array([0, 300], np.int32)
    banner("cell list unwrapped positions")
    for mode in (CELLS, PAIRS):
        _check(_build(_model(4.0), pos, cell, offsets, mode), pos, cell, offsets, 4.0)


def test_dense_cell_beyond_the_sort_capacity():
    """64 atoms in a 4 A box with r_cut = 6: about 900 neighbours per centre, past the
    512 the cell-list write pass sorts; those centres go through the all-pairs kernel."""
    rng = np.random.default_rng(14)
    pos = (rng.random((64, 3)) * 4.0).astype(np.float32)
    cell = np.diag([4.0] * 3).astype(np.float32)[None]
    offsets = np.array([0, 64], np.int32)
    banner("cell list dense cell")
    got = _build(_model(6.0), pos, cell, offsets, CELLS)
    ne = _check(got, pos, cell, offsets, 6.0)
    assert np.diff(got["rowptr"]).min() > 512, ne


def test_mode_is_validated():
    from paper_2604_15821_amd import janus
    ctx = janus.Context(_model(4.0))
    try:
        for bad in (-1, 3):
            with pytest.raises(janus.JanusError) as ex:
                ctx.set_edge_builder(bad)
            assert ex.value.code == janus.JANUS_EINVAL
    finally:
        ctx.close()
