"""Seeded synthetic inputs for the MatRIS-MoE training step.

This module draws structures (cells, positions, species), model weights and
reference labels.  It holds none of the method's arithmetic: no neighbour
test, no basis, no routing, no model evaluation.  Both the HIP path (through
the Python binding) and the float64 oracle consume exactly the arrays it
returns, so the two sides see the same bytes.

The five workloads stand in for the paper's 473M-configuration training set
(Sec. "Overview of the problem", edge tokens as the unit of work; the dataset
spans molecules, crystals, catalysis and MOFs).  No item of that dataset is
reproduced: every structure is drawn from the distributions documented on
each ``Workload`` below.

Draw order per workload (all from ``np.random.default_rng(seed)``):
structure kinds and sizes -> boxes -> positions -> species -> weights in blob
order -> E_ref -> F_ref.
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass, field

import numpy as np

N_SPECIES = 89


@dataclass(frozen=True)
class ModelConfig:
    """Hyper-parameters of the invariant MoE message-passing potential.

    d: embedding width; n_rbf: Bessel functions; n_blocks: interaction blocks;
    n_experts / top_k / d_hidden: edge-MoE size (each expert d -> d_hidden -> d);
    r_cut: neighbour cutoff in Angstrom.  The three-body fields describe the
    optional angular term (triplets of bonds shorter than r_cut3).  The
    atom_moe fields describe the optional feature-update MoE of every block
    (atom tokens routed by element type; each expert d -> d_hidden_f -> d).
    w_E, w_F, w_S weigh the energy, force and stress terms of the loss (stress
    in eV/A^3; w_S = 0 leaves it out).  n_heads > 0 adds multi-head
    self-attention over every atom's edge messages (head width d / n_heads).
    n_tasks > 0 adds the task-aware embedding: per-structure task, charge and
    spin labels (indices below n_tasks, n_charges, n_spins) and the element
    composition each add a vector to the atom embedding.  robust = 1 replaces
    the mean-squared loss by the robust multi-task loss: per-structure Huber
    losses of width huber_delta, weighted by a soft threshold at robust_tau
    standard deviations of the structure's task.  route_feat = 1 adds a linear
    router on the evolving edge token to every edge MoE: logits
    (Pc[Z_i] + Pn[Z_j]) + X_e Wr + beta with Wr [d, E] per block.
    """

    d: int
    n_rbf: int
    n_blocks: int
    n_experts: int
    top_k: int
    d_hidden: int
    r_cut: float
    n_species: int = N_SPECIES
    env_p: int = 6
    three_body: bool = False
    r_cut3: float = 3.5
    n_experts3: int = 0
    top_k3: int = 0
    d_hidden3: int = 0
    n_legendre: int = 5
    w_E: float = 1.0
    w_F: float = 1.0
    atom_moe: bool = False
    n_experts_f: int = 0
    top_k_f: int = 0
    d_hidden_f: int = 0
    w_S: float = 0.0
    n_heads: int = 0
    n_tasks: int = 0
    n_charges: int = 0
    n_spins: int = 0
    robust: int = 0
    huber_delta: float = math.inf
    robust_tau: float = 2.0
    route_feat: int = 0

    def weight_shapes(self):
        """Named weight tensors in blob order, with the fan-in used at init.

        Returns a list of (name, shape, fan_in); fan_in None marks a one-hot
        table drawn N(0, 1) and 'zero' marks the fixed routing bias.
        """
        d, E, h, nb, S = self.d, self.n_experts, self.d_hidden, self.n_rbf, self.n_species
        out = [("A", (S, d), None)]
        if self.n_tasks:
            out += [("Tk", (self.n_tasks, d), None), ("Qe", (self.n_charges, d), None),
                    ("Se", (self.n_spins, d), None), ("Wc", (S, d), None)]
        for t in range(self.n_blocks):
            p = f"blocks.{t}."
            out += [
                (p + "W_b", (nb, d), nb),
                (p + "Pc", (S, E), None),
                (p + "Pn", (S, E), None),
                (p + "beta", (E,), "zero"),
            ]
            if self.route_feat:
                out += [(p + "Wr", (d, E), d)]
            out += [
                (p + "W1", (E, d, h), d),
                (p + "W2", (E, h, d), h),
            ]
            if self.three_body:
                E3, h3 = self.n_experts3, self.d_hidden3
                nf = self.n_legendre * nb
                out += [
                    (p + "W_a", (nf, d), nf),
                    (p + "P3a", (S, E3), None),
                    (p + "P3b", (S, E3), None),
                    (p + "P3c", (S, E3), None),
                    (p + "beta3", (E3,), "zero"),
                    (p + "W1a", (E3, d, h3), d),
                    (p + "W2a", (E3, h3, d), h3),
                ]
            if self.atom_moe:
                Ef, hf = self.n_experts_f, self.d_hidden_f
                out += [
                    (p + "Pf", (S, Ef), None),
                    (p + "betaf", (Ef,), "zero"),
                    (p + "W1f", (Ef, d, hf), d),
                    (p + "W2f", (Ef, hf, d), hf),
                ]
            if self.n_heads:
                out += [
                    (p + "Wqkv", (d, 3 * d), d),
                    (p + "Wo", (d, d), d),
                ]
        out += [("W_o1", (d, d), d), ("w_o2", (d,), d)]
        return out


@dataclass(frozen=True)
class Workload:
    """A synthetic batch recipe.

    kind 'cubic'  : n_struct cubic cells of n_atoms each at `density`.
    kind 'ortho'  : orthorhombic cells, sides proportional to (1, a, b) with
                    a, b ~ U[1, 1.5], volume n_atoms / density.
    kind 'mixed'  : n_struct structures, atom count round(exp(U[ln lo, ln hi])),
                    crystal with probability p_crystal (cubic cell at
                    `density`), otherwise a molecule: uniform in a sphere of
                    local density `mol_density`, centred in a cubic box of
                    side 2R + vacuum.
    zipf_s        : if > 0, block routing biases beta_x = -zipf_s * ln(rank_x)
                    with rank a seeded permutation of 1..E (skewed expert load).
    """

    name: str
    kind: str
    n_struct: int
    n_atoms: int
    density: float
    model: ModelConfig
    seed: int = 0
    size_lo: int = 8
    size_hi: int = 512
    p_crystal: float = 0.7
    mol_density: float = 0.02
    vacuum: float = 20.0
    zipf_s: float = 0.0


_M_TINY = ModelConfig(d=64, n_rbf=8, n_blocks=2, n_experts=4, top_k=1, d_hidden=128, r_cut=4.0)
_M_SMALL = ModelConfig(d=128, n_rbf=16, n_blocks=3, n_experts=8, top_k=2, d_hidden=512, r_cut=5.0)
_M_3B = dataclasses.replace(_M_SMALL, three_body=True, r_cut3=3.5, n_experts3=8, top_k3=2, d_hidden3=256)
_M_ATOM = dataclasses.replace(_M_SMALL, atom_moe=True, n_experts_f=8, top_k_f=2, d_hidden_f=512)
# stress weight 0.1 on stresses measured in GPa (1 eV/A^3 = 160.2177 GPa)
_M_STRESS = dataclasses.replace(_M_SMALL, w_S=0.1 * 160.2177 ** 2)
_M_ATTN = dataclasses.replace(_M_SMALL, n_heads=4)
# task-aware embedding: 4 datasets, total charges -2..2, spin multiplicities 1..4
_M_TASK = dataclasses.replace(_M_SMALL, n_tasks=4, n_charges=5, n_spins=4)
# robust multi-task loss (Huber width 1, down-weighting beyond 2 standard deviations per task)
_M_ROBUST = dataclasses.replace(_M_TASK, robust=1, huber_delta=1.0, robust_tau=2.0)
_M_BIG = ModelConfig(d=512, n_rbf=16, n_blocks=4, n_experts=64, top_k=2, d_hidden=2048, r_cut=6.0)
# attention over large neighbourhoods (about 110 edges per atom at 0.12 atoms / A^3), d = 256, 8 heads
_M_ATTN_WIDE = dataclasses.replace(_M_SMALL, d=256, n_heads=8, r_cut=6.0)
# four heads of 128 columns at d = 512 (the head count and width of the paper's larger
# models' attention) on the small batch's structures
_M_ATTN_H128 = dataclasses.replace(_M_SMALL, d=512, n_heads=4)
# routing on the evolving edge tokens (species tables plus a linear layer on X_e)
_M_FEAT = dataclasses.replace(_M_SMALL, route_feat=1)

WORKLOADS = {
    "tiny": Workload("tiny", "cubic", 8, 32, 0.08, _M_TINY),
    "small": Workload("small", "ortho", 64, 64, 0.08, _M_SMALL),
    "threebody": Workload("threebody", "ortho", 64, 64, 0.08, _M_3B),
    "atom_moe": Workload("atom_moe", "ortho", 64, 64, 0.08, _M_ATOM),
    "stress": Workload("stress", "ortho", 64, 64, 0.08, _M_STRESS),
    "attention": Workload("attention", "ortho", 64, 64, 0.08, _M_ATTN),
    "attention_wide": Workload("attention_wide", "ortho", 64, 64, 0.12, _M_ATTN_WIDE),
    "attention_h128": Workload("attention_h128", "ortho", 64, 64, 0.08, _M_ATTN_H128),
    "multitask": Workload("multitask", "ortho", 64, 64, 0.08, _M_TASK),
    "robust": Workload("robust", "ortho", 64, 64, 0.08, _M_ROBUST),
    "feature_routing": Workload("feature_routing", "ortho", 64, 64, 0.08, _M_FEAT),
    "shard": Workload("shard", "cubic", 256, 128, 0.1, _M_BIG),
    "irregular": Workload("irregular", "mixed", 512, 0, 0.1, _M_BIG, zipf_s=1.2),
}


@dataclass
class Batch:
    """One synthetic batch.  All float arrays are float32, ints int32."""

    pos: np.ndarray          # [N, 3] Cartesian positions, wrapped into the cell
    cell: np.ndarray         # [S, 3, 3] row vectors a, b, c (diagonal here)
    species: np.ndarray      # [N] atomic type index in 0..88
    offsets: np.ndarray      # [S+1] structure s owns atoms offsets[s]:offsets[s+1]
    E_ref: np.ndarray        # [S] per-atom reference energy of each structure
    F_ref: np.ndarray        # [N, 3]
    weights: dict = field(default_factory=dict)   # name -> float32 array
    S_ref: np.ndarray | None = None   # [S, 3, 3] reference stress (eV/A^3), symmetric
    task: np.ndarray | None = None    # [S] int32 labels of the task-aware embedding
    charge: np.ndarray | None = None  # [S] int32 index of the total charge
    spin: np.ndarray | None = None    # [S] int32 index of the spin multiplicity
    model: ModelConfig | None = None
    name: str = ""

    @property
    def n_atoms(self):
        return int(self.pos.shape[0])

    @property
    def n_struct(self):
        return int(self.cell.shape[0])


def _draw_weights(rng, m: ModelConfig, zipf_s: float):
    w = {}
    for name, shape, fan in m.weight_shapes():
        if fan == "zero":
            if zipf_s > 0:
                rank = rng.permutation(shape[0]) + 1
                w[name] = (-zipf_s * np.log(rank.astype(np.float64))).astype(np.float32)
            else:
                w[name] = np.zeros(shape, np.float32)
        elif fan is None:
            w[name] = rng.standard_normal(shape).astype(np.float32)
        else:
            w[name] = (rng.standard_normal(shape) / np.sqrt(fan)).astype(np.float32)
    return w


def make_batch(wl: Workload | str, seed: int | None = None, n_struct: int | None = None) -> Batch:
    """Draw one batch of workload `wl` (name or Workload).

    n_struct, if given, truncates the structure count (the draws for the kept
    structures are identical to those of the full batch only for the weights;
    use it for small test cases, not for sampling a full batch).
    """
    if isinstance(wl, str):
        wl = WORKLOADS[wl]
    rng = np.random.default_rng(wl.seed if seed is None else seed)
    S = wl.n_struct if n_struct is None else n_struct
    m = wl.model

    # 1. structure kinds and sizes
    if wl.kind == "mixed":
        crystal = rng.random(S) < wl.p_crystal
        sizes = np.rint(np.exp(rng.uniform(np.log(wl.size_lo), np.log(wl.size_hi), S))).astype(np.int64)
    else:
        crystal = np.ones(S, bool)
        sizes = np.full(S, wl.n_atoms, np.int64)

    # 2. boxes
    sides = np.zeros((S, 3))
    mol_R = np.zeros(S)
    if wl.kind == "ortho":
        ab = rng.uniform(1.0, 1.5, (S, 2))
        for s in range(S):
            a0 = (sizes[s] / wl.density / (ab[s, 0] * ab[s, 1])) ** (1.0 / 3.0)
            sides[s] = (a0, a0 * ab[s, 0], a0 * ab[s, 1])
    else:
        for s in range(S):
            if crystal[s]:
                sides[s] = (sizes[s] / wl.density) ** (1.0 / 3.0)
            else:
                mol_R[s] = (3.0 * sizes[s] / (4.0 * np.pi * wl.mol_density)) ** (1.0 / 3.0)
                sides[s] = 2.0 * mol_R[s] + wl.vacuum
    sides = sides.astype(np.float32)

    # 3. positions (fp32, wrapped into [0, L))
    pos = []
    for s in range(S):
        n = int(sizes[s])
        L = sides[s].astype(np.float64)
        if crystal[s]:
            p = rng.random((n, 3)) * L
        else:
            v = rng.standard_normal((n, 3))
            v /= np.linalg.norm(v, axis=1, keepdims=True)
            rad = mol_R[s] * rng.random(n) ** (1.0 / 3.0)
            p = 0.5 * L + v * rad[:, None]
        p = p.astype(np.float32)
        # rounding can land exactly on L; fold such coordinates back to 0
        p = np.where(p >= sides[s], np.float32(0.0), p)
        pos.append(p)
    pos = np.concatenate(pos, 0) if pos else np.zeros((0, 3), np.float32)

    # 4. species
    N = int(sizes.sum())
    species = rng.integers(0, m.n_species, N).astype(np.int32)

    # 5. weights, 6. references
    weights = _draw_weights(rng, m, wl.zipf_s)
    E_ref = rng.standard_normal(S).astype(np.float32)
    F_ref = rng.standard_normal((N, 3)).astype(np.float32)
    # 7. reference stresses: (a + a^T)/sqrt(2) GPa for a standard Gaussian a
    #    (off-diagonal variance 1 GPa^2, diagonal 2 GPa^2), stored in eV/A^3
    a = rng.standard_normal((S, 3, 3))
    S_ref = ((a + a.transpose(0, 2, 1)) / np.sqrt(2.0) / 160.2177).astype(np.float32)
    # 8. labels of the task-aware embedding (uniform over each label's range)
    labels = {}
    if m.n_tasks:
        labels = {"task": rng.integers(0, m.n_tasks, S).astype(np.int32),
                  "charge": rng.integers(0, m.n_charges, S).astype(np.int32),
                  "spin": rng.integers(0, m.n_spins, S).astype(np.int32)}

    cell = np.zeros((S, 3, 3), np.float32)
    for s in range(S):
        cell[s] = np.diag(sides[s])
    offsets = np.zeros(S + 1, np.int32)
    offsets[1:] = np.cumsum(sizes)
    return Batch(pos=pos, cell=cell, species=species, offsets=offsets, E_ref=E_ref,
                 F_ref=F_ref, weights=weights, model=m, name=wl.name, S_ref=S_ref, **labels)


def subset(batch: Batch, structs) -> Batch:
    """The sub-batch made of the listed structures (same weights)."""
    structs = list(structs)
    pos, spc, fref, sizes = [], [], [], []
    for s in structs:
        a, b = int(batch.offsets[s]), int(batch.offsets[s + 1])
        pos.append(batch.pos[a:b]); spc.append(batch.species[a:b]); fref.append(batch.F_ref[a:b])
        sizes.append(b - a)
    off = np.zeros(len(structs) + 1, np.int32)
    off[1:] = np.cumsum(sizes)
    return Batch(pos=np.concatenate(pos, 0), cell=batch.cell[structs].copy(),
                 species=np.concatenate(spc, 0), offsets=off, E_ref=batch.E_ref[structs].copy(),
                 F_ref=np.concatenate(fref, 0), weights=batch.weights, model=batch.model,
                 name=batch.name + "[sub]",
                 S_ref=None if batch.S_ref is None else batch.S_ref[structs].copy(),
                 **{k: None if getattr(batch, k) is None else getattr(batch, k)[structs].copy()
                    for k in ("task", "charge", "spin")})
