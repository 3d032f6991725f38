"""Neighbour list, reverse map and radial basis of the HIP path against the
oracle: edges bit-exact, basis to fp32 rounding."""
import numpy as np
import pytest

from helpers import banner, rel_l2

pytestmark = pytest.mark.gpu

# (workload, structures kept): several tiles and ragged tails, every geometry kind
GRAPH_CASES = [("tiny", None), ("small", 6), ("shard", 2), ("irregular", 24)]


def _ctx(model):
    from paper_2604_15821_amd import janus
    return janus.Context(model)


def _sub(name, n):
    from paper_2604_15821_amd.synth import make_batch, subset
    b = make_batch(name)
    return b if n is None else subset(b, range(n))


@pytest.mark.parametrize("name,n", GRAPH_CASES)
def test_neighbor_list_is_bit_exact(name, n):
    import torch
    from oracle.neighbors import neighbor_list, reverse_map
    from paper_2604_15821_amd import janus
    b = _sub(name, n)
    banner("neighbor_list", name, n, b.n_atoms)
    d = janus.upload(b)
    ctx = _ctx(b.model)
    nl = ctx.build_edges(d["pos"], d["cell"], d["offsets"])
    torch.cuda.synchronize()
    ei, ej, sh, rp = neighbor_list(b.pos, b.cell, b.offsets, b.model.r_cut)
    rev = reverse_map(ei, ej, sh, b.n_atoms)
    assert nl.n_edges == ei.shape[0]
    assert (nl.ei.cpu().numpy() == ei).all()
    assert (nl.ej.cpu().numpy() == ej).all()
    assert (nl.shift.cpu().numpy() == sh).all()
    assert (nl.rowptr.cpu().numpy() == rp).all()
    assert (nl.rev.cpu().numpy() == rev).all()
    ctx.close()


def test_capacity_two_call_pattern_and_rebuild():
    import torch
    from paper_2604_15821_amd import janus
    b = _sub("tiny", 3)
    banner("capacity")
    d = janus.upload(b)
    ctx = _ctx(b.model)
    with pytest.raises(janus.JanusError) as ex:
        ctx.build_edges(d["pos"], d["cell"], d["offsets"], capacity=10)
    assert ex.value.code == janus.JANUS_ECAPACITY
    nl = ctx.build_edges(d["pos"], d["cell"], d["offsets"])
    n = ctx.build_edges_into(d["pos"], d["cell"], d["offsets"], nl)
    assert n == nl.n_edges
    ctx.close()


def test_bad_offsets_and_cells_are_rejected():
    import torch
    from paper_2604_15821_amd import janus
    b = _sub("tiny", 2)
    banner("bad inputs")
    d = janus.upload(b)
    ctx = _ctx(b.model)
    bad = d["offsets"].clone()
    bad[1] = 1000
    with pytest.raises(janus.JanusError) as ex:
        ctx.build_edges(d["pos"], d["cell"], bad)
    assert ex.value.code == janus.JANUS_EINVAL
    cell = d["cell"].clone()
    cell[0, 0, 1] = 0.5
    with pytest.raises(janus.JanusError) as ex:
        ctx.build_edges(d["pos"], cell, d["offsets"])
    assert ex.value.code == janus.JANUS_EUNSUPPORTED
    ctx.close()


@pytest.mark.parametrize("name,n", [("tiny", None), ("small", 3)])
def test_basis_matches_oracle(name, n):
    import torch
    from oracle.model import build_graph
    from paper_2604_15821_amd import janus
    b = _sub(name, n)
    banner("basis", name)
    d = janus.upload(b)
    ctx = _ctx(b.model)
    nl = ctx.build_edges(d["pos"], d["cell"], d["offsets"])
    m = b.model
    T, k, Ne = m.n_blocks, m.top_k, nl.n_edges
    dbg = {"basis": torch.empty(Ne * m.n_rbf, device="cuda:0")}
    ctx.step(d["pos"], d["cell"], d["species"], d["offsets"], nl, d["W"], d["E_ref"], d["F_ref"], debug=dbg)
    torch.cuda.synchronize()
    g = build_graph(b.pos, b.cell, b.offsets, m.r_cut, m.n_rbf)
    got = dbg["basis"].cpu().numpy().reshape(Ne, m.n_rbf)
    assert np.abs(got - g.B).max() <= 1e-6 * max(1.0, np.abs(g.B).max())
    ctx.close()
