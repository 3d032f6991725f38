"""Task-aware embedding (task, charge, spin, element composition) on the GPU
(janus_step_ex) against the float64 oracle: energy 1e-5, loss 1e-5, forces
and every weight gradient (the four tables included) 1e-3 relative L2; the
same with every optional term of the model switched on at once; missing or
out-of-range labels are rejected."""
import dataclasses

import numpy as np
import pytest

from helpers import TOL_E, TOL_F, TOL_LOSS, TOL_W, banner, energy_error, rel_l2

pytestmark = pytest.mark.gpu

FIXED = ("beta", "beta3", "betaf")


def _batch(name):
    from paper_2604_15821_amd.synth import _draw_weights, make_batch, subset
    if name == "multitask-4":
        return subset(make_batch("multitask"), range(4))
    if name == "everything":
        # bond angles, feature-update MoE, attention, stress and the task-aware embedding
        b = subset(make_batch("threebody"), range(2))
        m = dataclasses.replace(b.model, d=64, d_hidden=128, n_experts=4, n_experts3=3, d_hidden3=64, n_rbf=8,
                                n_blocks=2, atom_moe=True, n_experts_f=3, top_k_f=2, d_hidden_f=64,
                                w_S=0.1 * 160.2177 ** 2, n_heads=2, n_tasks=3, n_charges=5, n_spins=2)
        rng = np.random.default_rng(21)
        return dataclasses.replace(b, model=m, weights=_draw_weights(rng, m, 0.0),
                                   task=np.array([2, 0], np.int32), charge=np.array([1, 4], np.int32),
                                   spin=np.array([1, 0], np.int32))
    raise KeyError(name)


def _run(b, labels="batch"):
    import torch
    from paper_2604_15821_amd import janus
    d = janus.upload(b)
    ctx = janus.Context(b.model)
    try:
        nl = ctx.build_edges(d["pos"], d["cell"], d["offsets"])
        lab = d["labels"] if labels == "batch" else labels
        loss, E, F, dW = ctx.step(d["pos"], d["cell"], d["species"], d["offsets"], nl, d["W"], d["E_ref"],
                                  d["F_ref"], S_ref=d["S_ref"] if b.model.w_S else None, labels=lab)
        torch.cuda.synchronize()
        return float(loss.cpu()[0]), E.cpu().numpy(), F.cpu().numpy(), dW.cpu().numpy()
    finally:
        ctx.close()


@pytest.fixture(scope="module", params=["multitask-4", "everything"])
def case(request):
    from oracle.model import Params, build_graph_for, forward_energy, training_step
    b = _batch(request.param)
    banner("multitask", request.param, b.n_struct, "structures", b.n_atoms, "atoms")
    loss, E, F, grad, aux = training_step(b, return_aux=True)
    _, cache = forward_energy(b.species, aux["graph"], Params.from_weights(b.weights, b.model), aux["routing"])
    return b, _run(b), (loss, E, F, grad, cache)


def test_energy_loss_forces(case):
    b, (g_loss, g_E, g_F, g_W), (loss, E, F, grad, cache) = case
    err, ferr = energy_error(g_E, E, cache["eps"], b.offsets), rel_l2(g_F, F)
    print(f"  energy error {err:.2e}, force rel L2 {ferr:.2e}", flush=True)
    assert err <= TOL_E
    assert abs(g_loss - loss) <= TOL_LOSS * abs(loss)
    assert ferr <= TOL_F


def test_weight_gradients(case):
    from paper_2604_15821_amd import janus
    b, (g_loss, g_E, g_F, g_W), (loss, E, F, grad, cache) = case
    got = janus.unpack(g_W, b.model)
    worst = {}
    for name, ref in grad.items():
        if name.rsplit(".", 1)[-1] in FIXED:
            assert not got[name].any(), name
            continue
        if not ref.any():
            assert not got[name].any(), name
            continue
        worst[name] = rel_l2(got[name], ref)
    print("  tables", {k: f"{worst[k]:.1e}" for k in ("Tk", "Qe", "Se", "Wc") if k in worst}, flush=True)
    assert max(worst.values()) <= TOL_W, {k: v for k, v in worst.items() if v > TOL_W}


def test_missing_or_bad_labels_are_rejected():
    import torch
    from paper_2604_15821_amd import janus
    b = _batch("multitask-4")
    banner("multitask labels rejected")
    with pytest.raises(janus.JanusError) as ex:
        _run(b, labels=None)
    assert ex.value.code == janus.JANUS_EINVAL
    bad = dataclasses.replace(b, spin=np.array([0, 1, 4, 2], np.int32))     # 4 spin levels: index 4 is out
    with pytest.raises(janus.JanusError) as ex:
        _run(bad)
    assert ex.value.code == janus.JANUS_EINVAL
