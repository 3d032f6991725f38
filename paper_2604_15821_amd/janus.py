"""Thin ctypes binding of libjanus (argument marshalling only).

Every computation runs in the HIP library; PyTorch is used here only to
allocate device memory and to pick the stream.  Importing this module loads
the in-tree ``_lib/libjanus.so`` and raises if it has not been built: there
is no CPU fallback.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "_lib", "libjanus.so")

JANUS_OK, JANUS_EINVAL, JANUS_ECAPACITY, JANUS_ENOMEM, JANUS_EHIP, JANUS_EUNSUPPORTED = 0, -1, -2, -3, -4, -5


class JanusError(RuntimeError):
    def __init__(self, code, where):
        self.code = code
        super().__init__(f"{where}: {_lib().janus_strerror(code).decode()} (code {code})")


class Config(C.Structure):
    _fields_ = [
        ("n_species", C.c_int32), ("d", C.c_int32), ("n_rbf", C.c_int32), ("n_blocks", C.c_int32),
        ("n_experts", C.c_int32), ("top_k", C.c_int32), ("d_hidden", C.c_int32), ("env_p", C.c_int32),
        ("r_cut", C.c_float), ("three_body", C.c_int32), ("r_cut3", C.c_float), ("n_experts3", C.c_int32),
        ("top_k3", C.c_int32), ("d_hidden3", C.c_int32), ("n_legendre", C.c_int32), ("w_E", C.c_float),
        ("w_F", C.c_float), ("atom_moe", C.c_int32), ("n_experts_f", C.c_int32), ("top_k_f", C.c_int32),
        ("d_hidden_f", C.c_int32), ("w_S", C.c_float), ("n_heads", C.c_int32), ("n_tasks", C.c_int32),
        ("n_charges", C.c_int32), ("n_spins", C.c_int32), ("robust", C.c_int32), ("huber_delta", C.c_float),
        ("robust_tau", C.c_float), ("route_feat", C.c_int32),
    ]


class TensorDesc(C.Structure):
    _fields_ = [("name", C.c_char * 48), ("offset", C.c_int64), ("ndim", C.c_int32), ("shape", C.c_int64 * 3)]


class Edges(C.Structure):
    _fields_ = [("n_edges", C.c_int64), ("ei", C.c_void_p), ("ej", C.c_void_p), ("shift", C.c_void_p),
                ("rowptr", C.c_void_p), ("rev", C.c_void_p)]


class Labels(C.Structure):
    _fields_ = [("task", C.c_void_p), ("charge", C.c_void_p), ("spin", C.c_void_p)]


class ProfileEntry(C.Structure):
    _fields_ = [("name", C.c_char * 32), ("launches", C.c_int64), ("ms", C.c_double), ("flops", C.c_double),
                ("bytes", C.c_double)]


class Debug(C.Structure):
    _fields_ = [("eid", C.c_void_p), ("gate", C.c_void_p), ("counts", C.c_void_p), ("pos", C.c_void_p),
                ("basis", C.c_void_p), ("tri_e", C.c_void_p), ("tri_e2", C.c_void_p), ("eid3", C.c_void_p),
                ("gate3", C.c_void_p), ("eidf", C.c_void_p), ("gatef", C.c_void_p), ("gap", C.c_void_p)]

    KEYS = ("eid", "gate", "counts", "pos", "basis", "tri_e", "tri_e2", "eid3", "gate3", "eidf", "gatef", "gap")


_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"libjanus is not built ({LIB_PATH}); run paper_2604_15821_amd.build")
        # PyTorch's HIP runtime must be in the process before the library is: loaded
        # first, the library would bring in a second runtime (its link-time one), and
        # device memory of one runtime is not valid in the other
        import torch  # noqa: F401
        lib = C.CDLL(LIB_PATH)
        vp, i32, i64 = C.c_void_p, C.c_int32, C.c_int64
        lib.janus_strerror.restype = C.c_char_p
        lib.janus_strerror.argtypes = [C.c_int]
        lib.janus_create.argtypes = [C.POINTER(Config), C.POINTER(vp)]
        lib.janus_destroy.argtypes = [vp]
        lib.janus_destroy.restype = None
        lib.janus_weight_layout.argtypes = [C.POINTER(Config), C.POINTER(TensorDesc), C.POINTER(i32), C.POINTER(i64)]
        lib.janus_build_edges.argtypes = [vp, vp, vp, vp, i32, i32, i64, vp, vp, vp, vp, vp, C.POINTER(i64), vp]
        lib.janus_step.argtypes = [vp, vp, vp, vp, vp, i32, i32, C.POINTER(Edges), vp, vp, vp, vp, vp, vp, vp,
                                   C.POINTER(Debug), vp]
        lib.janus_step_stress.argtypes = [vp, vp, vp, vp, vp, i32, i32, C.POINTER(Edges), vp, vp, vp, vp, vp, vp,
                                          vp, vp, vp, C.POINTER(Debug), vp]
        lib.janus_step_ex.argtypes = [vp, vp, vp, vp, vp, i32, i32, C.POINTER(Edges), vp, vp, vp, vp,
                                      C.POINTER(Labels), vp, vp, vp, vp, vp, C.POINTER(Debug), vp]
        lib.janus_step_pos.argtypes = [vp, vp, vp, vp, vp, i32, i32, C.POINTER(Edges), vp, vp, vp, vp,
                                       C.POINTER(Labels), vp, vp, vp, vp, vp, vp, C.POINTER(Debug), vp]
        lib.janus_grouped_gemm.argtypes = [vp, vp, vp, vp, vp, i32, i64, i32, i32, i32, vp]
        lib.janus_grouped_wgrad.argtypes = [vp, vp, vp, vp, vp, i32, i64, i32, i32, vp]
        lib.janus_grouped_gemm_noalloc.argtypes = [vp, vp, vp, vp, i32, i64, i32, i32, i32, vp]
        lib.janus_wgrad_chunk_rows.argtypes = [i64, i32, i32]
        lib.janus_wgrad_chunk_rows.restype = i32
        lib.janus_set_workspace_limit.argtypes = [vp, i64]
        lib.janus_set_concurrency.argtypes = [vp, C.c_int]
        lib.janus_set_edge_builder.argtypes = [vp, C.c_int32]
        lib.janus_last_chunks.argtypes = [vp]
        lib.janus_last_triplets.argtypes = [vp]
        lib.janus_last_triplets.restype = i64
        lib.janus_profile_enable.argtypes = [vp, C.c_int]
        lib.janus_profile_read.argtypes = [vp, C.POINTER(ProfileEntry), i32]
        _LIB = lib
    return _LIB


def exported_symbols():
    """Names the library exports (checked against include/janus.h by the CPU tests)."""
    lib = _lib()
    names = ["janus_create", "janus_destroy", "janus_weight_layout", "janus_build_edges", "janus_step",
             "janus_step_stress", "janus_step_ex", "janus_step_pos",
             "janus_grouped_gemm", "janus_grouped_gemm_noalloc", "janus_grouped_wgrad", "janus_wgrad_chunk_rows",
             "janus_profile_enable",
             "janus_profile_read",
             "janus_set_workspace_limit", "janus_set_concurrency", "janus_set_edge_builder", "janus_last_chunks",
             "janus_last_triplets", "janus_strerror"]
    return [n for n in names if hasattr(lib, n)]


def wgrad_chunk_rows(M: int, P: int, Q: int) -> int:
    """Row-chunk length of the weight-gradient contraction over M rows into P x Q blocks."""
    r = int(_lib().janus_wgrad_chunk_rows(int(M), int(P), int(Q)))
    if r < 0:
        raise JanusError(r, "janus_wgrad_chunk_rows")
    return r


def make_config(model) -> Config:
    """Config from a ModelConfig-like object (attribute names as in the C struct)."""
    c = Config()
    for name, _ in Config._fields_:
        v = getattr(model, name)
        setattr(c, name, int(v) if not isinstance(v, float) else v)
    return c


def weight_layout(model):
    """[(name, offset, shape)] and the blob size, from the library."""
    lib = _lib()
    cfg = make_config(model)
    n = C.c_int32(0)
    tot = C.c_int64(0)
    rc = lib.janus_weight_layout(C.byref(cfg), None, C.byref(n), C.byref(tot))
    if rc:
        raise JanusError(rc, "janus_weight_layout")
    descs = (TensorDesc * n.value)()
    rc = lib.janus_weight_layout(C.byref(cfg), descs, C.byref(n), C.byref(tot))
    if rc:
        raise JanusError(rc, "janus_weight_layout")
    out = [(d.name.decode(), int(d.offset), tuple(int(d.shape[k]) for k in range(d.ndim))) for d in descs]
    return out, int(tot.value)


def pack_weights(weights: dict, model) -> np.ndarray:
    layout, total = weight_layout(model)
    blob = np.zeros(total, np.float32)
    for name, off, shape in layout:
        w = np.asarray(weights[name], np.float32)
        if w.shape != shape:
            raise ValueError(f"{name}: shape {w.shape} != {shape}")
        blob[off:off + w.size] = w.reshape(-1)
    return blob


def unpack(blob: np.ndarray, model) -> dict:
    layout, _ = weight_layout(model)
    return {name: blob[off:off + int(np.prod(shape))].reshape(shape) for name, off, shape in layout}


def _ptr(t):
    return C.c_void_p(0 if t is None else t.data_ptr())


_DTYPES = {"f32": "float32", "i32": "int32", "i8": "int8"}


def _arg(t, name, kind, shape=None, device=None, optional=False):
    """Check one tensor argument before its address goes to the library: the
    library reads raw memory, so a wrong dtype, a strided view, a host tensor or
    a wrong size would be misread rather than rejected.  `shape` may use None
    for a free dimension; returns the tensor."""
    if t is None:
        if optional:
            return None
        raise ValueError(f"{name}: required")
    import torch
    want = getattr(torch, _DTYPES[kind])
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch tensor, got {type(t).__name__}")
    if t.dtype != want:
        raise TypeError(f"{name}: dtype {t.dtype}, expected {want}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if not t.is_cuda:
        raise ValueError(f"{name}: must be a device tensor (got {t.device})")
    if device is not None and t.device != device:
        raise ValueError(f"{name}: on {t.device}, expected {device}")
    if shape is not None:
        if t.dim() != len(shape) or any(w is not None and int(n) != int(w) for n, w in zip(t.shape, shape)):
            raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t


def _stream():
    import torch
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


@dataclass
class NeighborList:
    n_edges: int
    ei: object
    ej: object
    shift: object
    rowptr: object
    rev: object

    def as_struct(self) -> Edges:
        return Edges(self.n_edges, _ptr(self.ei).value, _ptr(self.ej).value, _ptr(self.shift).value,
                     _ptr(self.rowptr).value, _ptr(self.rev).value)


class Context:
    """A libjanus context on the current device."""

    def __init__(self, model):
        import torch
        # PyTorch carries its own HIP runtime next to the library's; when the library's
        # initialises first, PyTorch's then finds no device, so PyTorch goes first
        if torch.cuda.is_available():
            torch.cuda.current_device()
        self.model = model
        self.cfg = make_config(model)
        h = C.c_void_p()
        rc = _lib().janus_create(C.byref(self.cfg), C.byref(h))
        if rc:
            raise JanusError(rc, "janus_create")
        self.h = h
        self.n_weights = weight_layout(model)[1]
        self.capacity = 0
        self._nl_bufs = None

    def close(self):
        if self.h:
            import torch
            torch.cuda.synchronize()
            _lib().janus_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---------------------------------------------------------------- edges
    def build_edges(self, pos, cell, offsets, capacity=None) -> NeighborList:
        """Neighbour list of device tensors pos [N,3] f32, cell [S,3,3] f32, offsets [S+1] i32."""
        import torch
        dev = pos.device
        N = pos.shape[0]
        S = cell.shape[0]
        self._check_geometry(pos, cell, offsets)
        rowptr = torch.empty(N + 1, dtype=torch.int32, device=dev)
        ne = C.c_int64(0)
        cap = int(capacity if capacity is not None else max(self.capacity, 1))
        for _ in range(2):
            ei = torch.empty(cap, dtype=torch.int32, device=dev)
            ej = torch.empty(cap, dtype=torch.int32, device=dev)
            rev = torch.empty(cap, dtype=torch.int32, device=dev)
            sh = torch.empty(cap * 3, dtype=torch.int8, device=dev)
            rc = _lib().janus_build_edges(self.h, _ptr(pos), _ptr(cell), _ptr(offsets), N, S, cap, _ptr(ei), _ptr(ej),
                                          _ptr(sh), _ptr(rowptr), _ptr(rev), C.byref(ne), _stream())
            if rc == JANUS_ECAPACITY and capacity is None:
                cap = int(ne.value)
                self.capacity = cap
                continue
            if rc:
                raise JanusError(rc, "janus_build_edges")
            n = int(ne.value)
            return NeighborList(n, ei[:n], ej[:n], sh[:3 * n].view(n, 3) if n else sh[:0].view(0, 3), rowptr,
                                rev[:n])
        raise RuntimeError("edge capacity did not converge")

    def build_edges_into(self, pos, cell, offsets, nl: NeighborList):
        """Rebuild into existing buffers (capacity = their size); returns the edge count."""
        ne = C.c_int64(0)
        cap = int(nl.ei.shape[0])
        self._check_geometry(pos, cell, offsets)
        self._check_edges(nl, pos.shape[0], pos.device, room=True)
        rc = _lib().janus_build_edges(self.h, _ptr(pos), _ptr(cell), _ptr(offsets), pos.shape[0], cell.shape[0],
                                      cap, _ptr(nl.ei), _ptr(nl.ej), _ptr(nl.shift), _ptr(nl.rowptr), _ptr(nl.rev),
                                      C.byref(ne), _stream())
        if rc:
            raise JanusError(rc, "janus_build_edges")
        return int(ne.value)

    # ------------------------------------------------------- argument checks
    @staticmethod
    def _check_geometry(pos, cell, offsets):
        dev = pos.device
        _arg(pos, "pos", "f32", (None, 3))
        _arg(cell, "cell", "f32", (None, 3, 3), dev)
        _arg(offsets, "offsets", "i32", (cell.shape[0] + 1,), dev)

    @staticmethod
    def _check_edges(nl, N, dev, room=False):
        """Edge arrays of a neighbour list: [Ne] each ([capacity] with room=True: the
        buffers a rebuild writes into), shift [Ne, 3], rowptr [N+1]."""
        n = int(nl.ei.shape[0]) if room else nl.n_edges
        _arg(nl.rowptr, "nl.rowptr", "i32", (N + 1,), dev)
        for name, t in (("nl.ei", nl.ei), ("nl.ej", nl.ej), ("nl.rev", nl.rev)):
            _arg(t, name, "i32", (n,), dev)
        sh = nl.shift.reshape(-1) if nl.shift is not None and nl.shift.is_contiguous() else nl.shift
        _arg(sh, "nl.shift", "i8", (3 * n,), dev)

    def _check_step(self, pos, cell, species, offsets, nl, W, E_ref, F_ref, out, S_ref, stress, labels):
        m = self.model
        dev = pos.device
        self._check_geometry(pos, cell, offsets)
        N, S = pos.shape[0], cell.shape[0]
        _arg(species, "species", "i32", (N,), dev)
        self._check_edges(nl, N, dev)
        total = self.n_weights
        _arg(W, "W", "f32", (total,), dev)
        _arg(E_ref, "E_ref", "f32", (S,), dev)
        _arg(F_ref, "F_ref", "f32", (N, 3), dev)
        # a missing S_ref (with w_S > 0) or missing labels (with n_tasks > 0) is the library's
        # JANUS_EINVAL; only the layout of what is passed is checked here
        _arg(S_ref, "S_ref", "f32", (S, 3, 3), dev, optional=True)
        _arg(stress, "stress", "f32", (S, 3, 3), dev, optional=True)
        if out is not None:
            loss, E, F, dW = out
            _arg(loss, "loss", "f32", (1,), dev)
            _arg(E, "E", "f32", (S,), dev)
            _arg(F, "F", "f32", (N, 3), dev)
            _arg(dW, "dLdW", "f32", (total,), dev)
        if labels is not None:
            for name, t in zip(("task", "charge", "spin"), labels):
                _arg(t, f"labels.{name}", "i32", (S,), dev)

    # ----------------------------------------------------------------- step
    def step(self, pos, cell, species, offsets, nl: NeighborList, W, E_ref, F_ref, out=None, debug=None,
             S_ref=None, stress=None, labels=None, dLdR=None):
        """One training step; returns (loss [1], E [S], F [N,3], dLdW [like W]) device tensors.

        With S_ref [S,3,3] (needed when the model's w_S > 0) or a stress output
        tensor [S,3,3], writes the stress into `stress`; labels = (task, charge,
        spin) int32 device tensors [S] (needed when the model has n_tasks > 0);
        with a dLdR tensor [N,3], also writes the loss gradient in the positions."""
        import torch
        dev = pos.device
        N = pos.shape[0]
        S = cell.shape[0]
        self._check_step(pos, cell, species, offsets, nl, W, E_ref, F_ref, out, S_ref, stress, labels)
        if out is None:
            out = (torch.empty(1, dtype=torch.float32, device=dev), torch.empty(S, dtype=torch.float32, device=dev),
                   torch.empty(N, 3, dtype=torch.float32, device=dev), torch.empty_like(W))
        loss, E, F, dW = out
        edges = nl.as_struct()
        dbg = None
        if debug is not None:
            dbg = Debug(*[_ptr(debug.get(k)).value for k in Debug.KEYS])
        dbgp = C.byref(dbg) if dbg is not None else None
        _arg(dLdR, "dLdR", "f32", (N, 3), dev, optional=True)
        if dLdR is not None:
            lab = Labels(*[_ptr(x).value for x in labels]) if labels is not None else None
            rc = _lib().janus_step_pos(self.h, _ptr(pos), _ptr(cell), _ptr(species), _ptr(offsets), N, S,
                                       C.byref(edges), _ptr(W), _ptr(E_ref), _ptr(F_ref), _ptr(S_ref),
                                       C.byref(lab) if lab is not None else None, _ptr(loss), _ptr(E), _ptr(F),
                                       _ptr(stress), _ptr(dW), _ptr(dLdR), dbgp, _stream())
        elif S_ref is None and stress is None and labels is None:
            rc = _lib().janus_step(self.h, _ptr(pos), _ptr(cell), _ptr(species), _ptr(offsets), N, S, C.byref(edges),
                                   _ptr(W), _ptr(E_ref), _ptr(F_ref), _ptr(loss), _ptr(E), _ptr(F), _ptr(dW), dbgp,
                                   _stream())
        elif labels is None:
            rc = _lib().janus_step_stress(self.h, _ptr(pos), _ptr(cell), _ptr(species), _ptr(offsets), N, S,
                                          C.byref(edges), _ptr(W), _ptr(E_ref), _ptr(F_ref), _ptr(S_ref), _ptr(loss),
                                          _ptr(E), _ptr(F), _ptr(stress), _ptr(dW), dbgp, _stream())
        else:
            lab = Labels(*[_ptr(x).value for x in labels])
            rc = _lib().janus_step_ex(self.h, _ptr(pos), _ptr(cell), _ptr(species), _ptr(offsets), N, S,
                                      C.byref(edges), _ptr(W), _ptr(E_ref), _ptr(F_ref), _ptr(S_ref), C.byref(lab),
                                      _ptr(loss), _ptr(E), _ptr(F), _ptr(stress), _ptr(dW), dbgp, _stream())
        if rc:
            raise JanusError(rc, "janus_step")
        return loss, E, F, dW

    # ------------------------------------------------------------ workspace
    def set_workspace_limit(self, nbytes: int):
        rc = _lib().janus_set_workspace_limit(self.h, int(nbytes))
        if rc:
            raise JanusError(rc, "janus_set_workspace_limit")

    def set_concurrency(self, on: bool):
        """Expert weight gradients on the context's second stream (True) or on the caller's (False, the default)."""
        rc = _lib().janus_set_concurrency(self.h, int(bool(on)))
        if rc:
            raise JanusError(rc, "janus_set_concurrency")

    def set_edge_builder(self, mode: int):
        """Candidate search of build_edges: 0 automatic, 1 cell list everywhere, 2 all pairs everywhere."""
        rc = _lib().janus_set_edge_builder(self.h, int(mode))
        if rc:
            raise JanusError(rc, "janus_set_edge_builder")

    def last_chunks(self) -> int:
        return int(_lib().janus_last_chunks(self.h))

    def last_triplets(self) -> int:
        return int(_lib().janus_last_triplets(self.h))

    # ------------------------------------------------------------- profiler
    PROFILE_FAMILIES = ["expert_gemm", "expert_wgrad", "dense_gemm", "edge", "atom", "route", "graph", "other",
                        "attention"]

    def profile(self, on: bool, families=None):
        """Start (on) or stop the event profiler; `families` restricts it to some kernel families."""
        mask = 0
        if on:
            mask = -1 if families is None else sum(1 << self.PROFILE_FAMILIES.index(f) for f in families)
        rc = _lib().janus_profile_enable(self.h, mask)
        if rc:
            raise JanusError(rc, "janus_profile_enable")

    def profile_read(self) -> dict:
        """{family: {launches, ms, flops, bytes}} since profile(True) or the last read."""
        buf = (ProfileEntry * 16)()
        n = _lib().janus_profile_read(self.h, buf, 16)
        if n < 0:
            raise JanusError(n, "janus_profile_read")
        return {buf[q].name.decode(): {"launches": int(buf[q].launches), "ms": float(buf[q].ms),
                                        "flops": float(buf[q].flops), "bytes": float(buf[q].bytes)}
                for q in range(n)}

    # ---------------------------------------------------------------- GEMMs
    def grouped_gemm(self, A, B, row_off, K, N, trans_b, out=None):
        import torch
        M = A.shape[0]
        dev = A.device
        G = row_off.shape[0] - 1
        _arg(A, "A", "f32", (M, K))
        _arg(B, "B", "f32", (G, N, K) if trans_b else (G, K, N), dev)
        _arg(row_off, "row_off", "i32", (G + 1,), dev)
        if out is None:
            out = torch.empty(M, N, dtype=torch.float32, device=A.device)
        _arg(out, "out", "f32", (M, N), dev)
        rc = _lib().janus_grouped_gemm(self.h, _ptr(A), _ptr(B), _ptr(out), _ptr(row_off), row_off.shape[0] - 1, M,
                                       K, N, int(trans_b), _stream())
        if rc:
            raise JanusError(rc, "janus_grouped_gemm")
        return out

    def grouped_wgrad(self, A, B, row_off, out=None):
        import torch
        M, P = A.shape
        Q = B.shape[1]
        G = row_off.shape[0] - 1
        dev = A.device
        _arg(A, "A", "f32", (M, P))
        _arg(B, "B", "f32", (M, Q), dev)
        _arg(row_off, "row_off", "i32", (G + 1,), dev)
        if out is None:
            out = torch.empty(G, P, Q, dtype=torch.float32, device=A.device)
        _arg(out, "out", "f32", (G, P, Q), dev)
        rc = _lib().janus_grouped_wgrad(self.h, _ptr(A), _ptr(B), _ptr(out), _ptr(row_off), G, M, P, Q, _stream())
        if rc:
            raise JanusError(rc, "janus_grouped_wgrad")
        return out


def grouped_gemm_noalloc(A, B, row_off, K, N, trans_b, out):
    """janus_grouped_gemm_noalloc on the current device: C = A x B_g per row group into
    the caller's `out`, with the tile table in the library's fixed scratch (no allocation)."""
    M = A.shape[0]
    dev = A.device
    G = row_off.shape[0] - 1
    _arg(A, "A", "f32", (M, K))
    _arg(B, "B", "f32", (G, N, K) if trans_b else (G, K, N), dev)
    _arg(row_off, "row_off", "i32", (G + 1,), dev)
    _arg(out, "out", "f32", (M, N), dev)
    rc = _lib().janus_grouped_gemm_noalloc(_ptr(A), _ptr(B), _ptr(out), _ptr(row_off), G, M, K, N, int(trans_b),
                                           _stream())
    if rc:
        raise JanusError(rc, "janus_grouped_gemm_noalloc")
    return out


def upload(batch, device="cuda:0"):
    """Device copies of a synthetic batch: dict with pos, cell, species, offsets, E_ref, F_ref, W."""
    import torch
    t = lambda a, dt: torch.as_tensor(np.ascontiguousarray(a)).to(device=device, dtype=dt)
    return {
        "pos": t(batch.pos, torch.float32),
        "cell": t(batch.cell, torch.float32),
        "species": t(batch.species, torch.int32),
        "offsets": t(batch.offsets, torch.int32),
        "E_ref": t(batch.E_ref, torch.float32),
        "F_ref": t(batch.F_ref, torch.float32),
        "S_ref": None if batch.S_ref is None else t(batch.S_ref, torch.float32),
        "labels": None if batch.task is None else tuple(t(getattr(batch, k), torch.int32)
                                                        for k in ("task", "charge", "spin")),
        "W": t(pack_weights(batch.weights, batch.model), torch.float32),
    }
