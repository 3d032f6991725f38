"""Model shapes that the five workloads do not reach, against the oracle:
embedding width 256 and 512 with the three-body term, top-k of 3 and 4,
expert counts that are not powers of two, hidden widths that leave a partial
64-column GEMM tile (192, 320), few Legendre orders and basis functions, the
largest Legendre order (8: the power-series coefficients of the angle features
are largest there),
Zipf-skewed routing on a crystal/molecule mix (empty experts), and the
feature-update MoE at top-k 1, 3 and 4 (alone, with the three-body term,
and with every expert chosen)."""
import numpy as np
import pytest

from helpers import TOL_E, TOL_F, TOL_LOSS, TOL_W, banner, energy_error, rel_l2

pytestmark = pytest.mark.gpu


def _configs():
    from paper_2604_15821_amd.synth import ModelConfig, Workload
    return {
        "d256-k3-E5-h192": Workload(
            "d256-k3", "cubic", 3, 24, 0.08,
            ModelConfig(d=256, n_rbf=8, n_blocks=2, n_experts=5, top_k=3, d_hidden=192, r_cut=4.5), seed=3),
        "d64-k4-E6-h320-zipf": Workload(
            "d64-k4", "mixed", 6, 0, 0.1,
            ModelConfig(d=64, n_rbf=12, n_blocks=1, n_experts=6, top_k=4, d_hidden=320, r_cut=4.0), seed=5,
            size_lo=6, size_hi=40, zipf_s=1.2),
        "3b-d256-k3-L3": Workload(
            "3b-d256", "cubic", 2, 32, 0.08,
            ModelConfig(d=256, n_rbf=8, n_blocks=1, n_experts=3, top_k=1, d_hidden=128, r_cut=5.0, three_body=True,
                        r_cut3=3.5, n_experts3=5, top_k3=3, d_hidden3=192, n_legendre=3), seed=7),
        "3b-d512-k4-L4": Workload(
            "3b-d512", "cubic", 1, 32, 0.08,
            ModelConfig(d=512, n_rbf=8, n_blocks=1, n_experts=2, top_k=2, d_hidden=64, r_cut=5.0, three_body=True,
                        r_cut3=3.5, n_experts3=4, top_k3=4, d_hidden3=64, n_legendre=4), seed=11),
        "3b-d128-L8": Workload(
            "3b-L8", "cubic", 2, 32, 0.08,
            ModelConfig(d=128, n_rbf=8, n_blocks=1, n_experts=3, top_k=2, d_hidden=128, r_cut=5.0, three_body=True,
                        r_cut3=3.5, n_experts3=3, top_k3=2, d_hidden3=64, n_legendre=8), seed=23),
        "atom-d64-kf1-Ef5-hf192": Workload(
            "atom-d64", "cubic", 4, 20, 0.08,
            ModelConfig(d=64, n_rbf=8, n_blocks=2, n_experts=3, top_k=2, d_hidden=128, r_cut=4.5, atom_moe=True,
                        n_experts_f=5, top_k_f=1, d_hidden_f=192), seed=13),
        "3b-atom-d128-kf3-Ef6": Workload(
            "3b-atom", "cubic", 2, 24, 0.08,
            ModelConfig(d=128, n_rbf=8, n_blocks=2, n_experts=4, top_k=2, d_hidden=128, r_cut=4.5, three_body=True,
                        r_cut3=3.5, n_experts3=3, top_k3=2, d_hidden3=64, n_legendre=3, atom_moe=True,
                        n_experts_f=6, top_k_f=3, d_hidden_f=128), seed=17),
        "atom-d256-kf4-Ef4-hf320-zipf": Workload(
            "atom-zipf", "mixed", 5, 0, 0.1,
            ModelConfig(d=256, n_rbf=8, n_blocks=1, n_experts=6, top_k=2, d_hidden=64, r_cut=4.0, atom_moe=True,
                        n_experts_f=4, top_k_f=4, d_hidden_f=320), seed=19, size_lo=6, size_hi=30, zipf_s=1.2),
    }


@pytest.fixture(scope="module", params=list(_configs()))
def case(request):
    import torch
    from oracle.model import Params, forward_energy, training_step
    from paper_2604_15821_amd import janus
    from paper_2604_15821_amd.synth import make_batch
    wl = _configs()[request.param]
    b = make_batch(wl)
    banner("config", request.param, b.n_struct, "structures", b.n_atoms, "atoms")
    loss, E, F, grad, aux = training_step(b, return_aux=True)
    _, cache = forward_energy(b.species, aux["graph"], Params.from_weights(b.weights, b.model), aux["routing"])
    d = janus.upload(b)
    ctx = janus.Context(b.model)
    try:
        nl = ctx.build_edges(d["pos"], d["cell"], d["offsets"])
        gl, gE, gF, gW = ctx.step(d["pos"], d["cell"], d["species"], d["offsets"], nl, d["W"], d["E_ref"],
                                  d["F_ref"])
        torch.cuda.synchronize()
        out = {"loss": float(gl.cpu()[0]), "E": gE.cpu().numpy(), "F": gF.cpu().numpy(), "dW": gW.cpu().numpy(),
               "edges": nl.n_edges, "triplets": ctx.last_triplets()}
    finally:
        ctx.close()
    print(f"  {out['edges']} edges, {out['triplets']} triplets", flush=True)
    return b, out, (loss, E, F, grad, aux, cache)


def test_graph_sizes(case):
    b, out, (loss, E, F, grad, aux, cache) = case
    g = aux["graph"]
    assert out["edges"] == g.ei.size > 0
    assert out["triplets"] == (g.tri.te.size if g.tri is not None else 0)
    if b.model.three_body:
        assert out["triplets"] > 0


def test_energy_loss_forces(case):
    b, out, (loss, E, F, grad, aux, cache) = case
    err = energy_error(out["E"], E, cache["eps"], b.offsets)
    ferr = rel_l2(out["F"], F)
    print(f"  energy error {err:.2e}, force rel L2 {ferr:.2e}", flush=True)
    assert err <= TOL_E
    assert abs(out["loss"] - loss) <= TOL_LOSS * abs(loss)
    assert ferr <= TOL_F


def test_weight_gradients(case):
    from paper_2604_15821_amd import janus
    b, out, (loss, E, F, grad, aux, cache) = case
    got = janus.unpack(out["dW"], b.model)
    worst = 0.0
    for name, ref in grad.items():
        if name.rsplit(".", 1)[-1] in ("beta", "beta3", "betaf"):
            assert not got[name].any(), name
            continue
        if not ref.any():
            assert not got[name].any(), name
            continue
        e = rel_l2(got[name], ref)
        worst = max(worst, e)
        assert e <= TOL_W, (name, e)
    print(f"  worst per-tensor rel L2 {worst:.2e}", flush=True)
