"""Host-side checks of the C ABI: the library loads, exports every entry point
declared in include/janus.h, reports the weight layout the synthetic
generator uses, and rejects bad configurations before touching a GPU."""
import ctypes as C
import os
import re

import pytest
import torch  # noqa: F401  (PyTorch's HIP runtime first: the library then binds to it)

from paper_2604_15821_amd import janus
from paper_2604_15821_amd.synth import WORKLOADS, ModelConfig

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    txt = open(os.path.join(ROOT, "include", "janus.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(janus_[a-z_]+)\s*\(", txt)))


def test_library_exports_every_declared_entry_point():
    lib = C.CDLL(janus.LIB_PATH)
    names = _declared()
    assert len(names) >= 8
    for n in names:
        assert hasattr(lib, n), n


@pytest.mark.parametrize("name", list(WORKLOADS))
def test_weight_layout_matches_generator(name):
    m = WORKLOADS[name].model
    layout, total = janus.weight_layout(m)
    assert [(n, s) for n, _, s in layout] == [(n, s) for n, s, _ in m.weight_shapes()]
    off = 0
    for _, o, s in layout:
        assert o == off
        n = 1
        for x in s:
            n *= x
        off += n
    assert off == total


def test_pack_unpack_roundtrip():
    from paper_2604_15821_amd.synth import make_batch
    b = make_batch("tiny")
    blob = janus.pack_weights(b.weights, b.model)
    back = janus.unpack(blob, b.model)
    for k, v in b.weights.items():
        assert (back[k] == v).all()


@pytest.mark.parametrize("change,code", [
    (dict(d=96), janus.JANUS_EUNSUPPORTED),
    (dict(top_k=5), janus.JANUS_EINVAL),
    (dict(n_experts=65), janus.JANUS_EINVAL),
    (dict(env_p=5), janus.JANUS_EUNSUPPORTED),
    (dict(d_hidden=32), janus.JANUS_EINVAL),
    (dict(r_cut=0.0), janus.JANUS_EINVAL),
    (dict(robust=2), janus.JANUS_EINVAL),
    (dict(robust=1, huber_delta=0.0), janus.JANUS_EINVAL),
    (dict(robust=1, robust_tau=float("nan")), janus.JANUS_EINVAL),
    (dict(robust=1, n_tasks=300, n_charges=1, n_spins=1), janus.JANUS_EUNSUPPORTED),
    (dict(n_heads=4), janus.JANUS_EUNSUPPORTED),          # heads of 16 columns
    (dict(d=256, n_heads=1), janus.JANUS_EUNSUPPORTED),   # one head of 256 columns
    (dict(n_heads=3), janus.JANUS_EINVAL),                # does not divide d
])
def test_bad_configs_are_rejected_on_the_host(change, code):
    import dataclasses
    m = dataclasses.replace(WORKLOADS["tiny"].model, **change)
    cfg = janus.make_config(m)
    h = C.c_void_p()
    assert janus._lib().janus_create(C.byref(cfg), C.byref(h)) == code
    assert not h.value


def test_strerror_messages():
    lib = janus._lib()
    for code in (0, -1, -2, -3, -4, -5):
        assert lib.janus_strerror(code)
    assert b"unknown" in lib.janus_strerror(17)


def test_concurrency_switch_rejects_bad_arguments():
    lib = C.CDLL(janus.LIB_PATH)
    lib.janus_set_concurrency.argtypes = [C.c_void_p, C.c_int]
    assert lib.janus_set_concurrency(None, 1) == janus.JANUS_EINVAL


def test_binding_rejects_misfit_tensors_before_the_library():
    """The library reads raw memory, so the binding refuses a wrong dtype, a strided
    view or a host tensor instead of passing its address."""
    import torch
    pos = torch.zeros(4, 3)
    with pytest.raises(TypeError):
        janus._arg(pos.double(), "pos", "f32", (None, 3))
    with pytest.raises(TypeError):
        janus._arg(torch.zeros(3, dtype=torch.int64), "offsets", "i32", (3,))
    with pytest.raises(ValueError, match="contiguous"):
        janus._arg(torch.zeros(3, 4).t(), "pos", "f32", (None, 3))
    with pytest.raises(ValueError, match="device"):
        janus._arg(pos, "pos", "f32", (None, 3))
    with pytest.raises(ValueError, match="device"):
        janus.Context._check_geometry(pos, torch.zeros(1, 3, 3), torch.zeros(2, dtype=torch.int32))
    assert janus._arg(None, "stress", "f32", optional=True) is None
    with pytest.raises(ValueError):
        janus._arg(None, "W", "f32")


def test_wgrad_chunk_rule():
    """Chunk length of the weight-gradient contraction: 512 rows for the small batch's
    expert products (337,996 slot rows, 128 x 512 blocks: 2644 workgroups, where 256
    rows would double the partial tiles past half of the operand bytes), 2048 at the
    full-size expert shape (over a million rows, 512 x 2048 blocks), bounds 128 and 2048."""
    assert janus.wgrad_chunk_rows(337_996, 128, 512) == 512
    assert janus.wgrad_chunk_rows(1_200_000, 512, 2048) == 2048
    assert janus.wgrad_chunk_rows(2_000_000, 2048, 512) == 2048
    assert janus.wgrad_chunk_rows(20_000, 128, 512) == 512
    assert janus.wgrad_chunk_rows(100, 64, 64) == 2048
    assert janus.wgrad_chunk_rows(0, 64, 64) == 128
    with pytest.raises(janus.JanusError):
        janus.wgrad_chunk_rows(-1, 64, 64)
    with pytest.raises(janus.JanusError):
        janus.wgrad_chunk_rows(10, 0, 64)
