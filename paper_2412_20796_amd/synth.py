"""Seeded synthetic inputs: crystals, initial weights and targets.

This module holds no arithmetic of the model. It only draws random inputs with
the shapes and statistics of the paper's training data (MPtrj is not
available, so these stand in for it) and serves both the CPU oracle and the
GPU path, which must be fed identical inputs.

Workloads (atoms per cell, densities and cell shapes):

* ``cubic8``     - one cubic cell a = 4.0 A, 8 atoms.
* ``triclinic40``- 40 triclinic cells, lattice angles U(60, 120) deg,
                   atoms per cell log-uniform in [8, 64], density
                   U(0.07, 0.10) atoms/A^3.
* ``heavytail64``- 64 cells, atoms per cell round(24 exp(0.9 N(0,1))) clipped
                   to [2, 400], density U(0.06, 0.12) (the long-tailed size
                   distribution the paper reports for its dataset, Sec. III-C).
* ``super4096``  - one cubic supercell of 4096 atoms at density 0.085.
* ``wide128``    - 128 cells, atoms per cell log-uniform in [8, 128], density
                   U(0.07, 0.10), used with feature width 128 and 5 layers.

Positions are placed by random sequential addition of uniform fractional
coordinates, keeping every pair (periodic images included) at least 1.5 A
apart. Atomic numbers are uniform in 1..94. Positions are stored as fp32
Cartesian coordinates and the lattice (rows = lattice vectors) as fp32.

Random streams: ``numpy.random.default_rng([cfg, purpose, rep])`` with
purpose 0 = structures, 1 = weights, 2 = targets.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

N_ELEMENTS = 94
MIN_SEP = 1.5

WORKLOADS = {
    # name: (cfg id, model width, layers)
    "cubic8": (0, 64, 4),
    "triclinic40": (1, 64, 4),
    "heavytail64": (2, 64, 4),
    "super4096": (3, 64, 4),
    "wide128": (4, 128, 5),
}


@dataclass
class Batch:
    """Host-side batch of crystals (fp32 positions and lattices)."""

    atom_ptr: np.ndarray  # int32 [S+1]
    pos: np.ndarray  # float32 [N, 3], Cartesian, Angstrom
    lattice: np.ndarray  # float32 [S, 3, 3], rows are lattice vectors
    Z: np.ndarray  # int32 [N], 1..94

    @property
    def n_struct(self) -> int:
        return int(self.lattice.shape[0])

    @property
    def n_atoms(self) -> int:
        return int(self.pos.shape[0])


def _lattice_from_params(a, b, c, al, be, ga):
    """Standard orientation: a along x, b in the xy-plane."""
    ca, cb, cg = math.cos(al), math.cos(be), math.cos(ga)
    sg = math.sin(ga)
    ax = np.array([a, 0.0, 0.0])
    bx = np.array([b * cg, b * sg, 0.0])
    cx = c * cb
    cy = c * (ca - cb * cg) / sg
    cz = math.sqrt(max(c * c - cx * cx - cy * cy, 0.0))
    return np.stack([ax, bx, np.array([cx, cy, cz])])


def _shortest_vector(L):
    best = np.inf
    for n in np.ndindex(5, 5, 5):
        n = np.array(n) - 2
        if not n.any():
            continue
        best = min(best, float(np.linalg.norm(n @ L)))
    return best


def _random_lattice(rng, n_atoms, rho_lo, rho_hi):
    while True:
        al, be, ga = np.radians(rng.uniform(60.0, 120.0, size=3))
        ca, cb, cg = math.cos(al), math.cos(be), math.cos(ga)
        if 1 + 2 * ca * cb * cg - ca * ca - cb * cb - cg * cg < 0.3:
            continue
        b_over_a, c_over_a = rng.uniform(0.75, 1.33, size=2)
        rho = rng.uniform(rho_lo, rho_hi)
        L = _lattice_from_params(1.0, b_over_a, c_over_a, al, be, ga)
        vol1 = abs(np.linalg.det(L))
        scale = (n_atoms / rho / vol1) ** (1.0 / 3.0)
        L = L * scale
        if np.linalg.norm(L, axis=1).min() < MIN_SEP or _shortest_vector(L) < MIN_SEP:
            continue
        return L


def _place_atoms(rng, L, n_atoms, max_fail=100_000):
    """Random sequential addition with a periodic minimum separation."""
    vol = abs(np.linalg.det(L))
    h = vol / np.linalg.norm(np.cross(L[[1, 2, 0]], L[[2, 0, 1]]), axis=1)
    reach = np.ceil(MIN_SEP / h + 0.5).astype(int)
    imgs = np.array(
        [
            (i, j, k)
            for i in range(-reach[0], reach[0] + 1)
            for j in range(-reach[1], reach[1] + 1)
            for k in range(-reach[2], reach[2] + 1)
        ],
        dtype=np.float64,
    )
    shifts = imgs @ L  # [I, 3]
    frac = np.empty((n_atoms, 3))
    placed = 0
    fails = 0
    while placed < n_atoms:
        f = rng.uniform(0.0, 1.0, size=3)
        if placed:
            df = frac[:placed] - f
            df -= np.round(df)
            # an image closer than MIN_SEP needs |df_a + n_a| <= MIN_SEP / h_a
            near = np.all(np.abs(df) <= MIN_SEP / h + 1e-9, axis=1)
            if near.any():
                dx = df[near] @ L
                d2 = ((dx[:, None, :] + shifts[None, :, :]) ** 2).sum(-1)
                if d2.min() < MIN_SEP * MIN_SEP:
                    fails += 1
                    if fails >= max_fail:
                        return None
                    continue
        frac[placed] = f
        placed += 1
    return frac


def _structure(rng, n_atoms, L=None, rho=(0.07, 0.10)):
    while True:
        lat = L if L is not None else _random_lattice(rng, n_atoms, *rho)
        frac = _place_atoms(rng, lat, n_atoms)
        if frac is not None:
            return lat, frac


def _assemble(structs, Zs):
    atom_ptr = np.zeros(len(structs) + 1, dtype=np.int32)
    pos, lat = [], []
    for s, (L, frac) in enumerate(structs):
        L32 = L.astype(np.float32)
        # Cartesian positions are rounded once from the fp64 product.
        pos.append((frac @ L).astype(np.float32))
        lat.append(L32)
        atom_ptr[s + 1] = atom_ptr[s] + frac.shape[0]
    return Batch(
        atom_ptr=atom_ptr,
        pos=np.ascontiguousarray(np.concatenate(pos, axis=0)),
        lattice=np.ascontiguousarray(np.stack(lat)),
        Z=np.ascontiguousarray(np.concatenate(Zs).astype(np.int32)),
    )


def make_batch(name: str, rep: int = 0) -> Batch:
    """Build the seeded batch of the named workload."""
    cfg = WORKLOADS[name][0]
    rng = np.random.default_rng([cfg, 0, rep])
    structs, Zs = [], []
    if name == "cubic8":
        L = np.eye(3) * 4.0
        structs.append(_structure(rng, 8, L=L))
        Zs.append(rng.integers(1, N_ELEMENTS + 1, size=8))
    elif name == "super4096":
        a = (4096 / 0.085) ** (1.0 / 3.0)
        structs.append(_structure(rng, 4096, L=np.eye(3) * a))
        Zs.append(rng.integers(1, N_ELEMENTS + 1, size=4096))
    else:
        if name == "triclinic40":
            S, rho = 40, (0.07, 0.10)
            counts = [int(round(math.exp(rng.uniform(math.log(8), math.log(64))))) for _ in range(S)]
        elif name == "heavytail64":
            S, rho = 64, (0.06, 0.12)
            counts = [int(np.clip(round(24 * math.exp(0.9 * rng.standard_normal())), 2, 400)) for _ in range(S)]
        elif name == "wide128":
            S, rho = 128, (0.07, 0.10)
            counts = [int(round(math.exp(rng.uniform(math.log(8), math.log(128))))) for _ in range(S)]
        else:
            raise KeyError(name)
        for n in counts:
            structs.append(_structure(rng, n, rho=rho))
            Zs.append(rng.integers(1, N_ELEMENTS + 1, size=n))
    return _assemble(structs, Zs)


def make_custom_batch(lattices, fracs, Zs) -> Batch:
    """Batch from explicit fp64 lattices and fractional coordinates."""
    structs = [(np.asarray(L, dtype=np.float64), np.asarray(f, dtype=np.float64)) for L, f in zip(lattices, fracs)]
    return _assemble(structs, [np.asarray(z) for z in Zs])


def random_crystals(seed: int, n_struct: int, n_lo: int, n_hi: int, rho=(0.07, 0.10)) -> Batch:
    """Small random triclinic batch for tests (same recipe, free seed)."""
    rng = np.random.default_rng([99, 0, seed])
    structs, Zs = [], []
    for _ in range(n_struct):
        n = int(rng.integers(n_lo, n_hi + 1))
        structs.append(_structure(rng, n, rho=rho))
        Zs.append(rng.integers(1, N_ELEMENTS + 1, size=n))
    return _assemble(structs, Zs)


def boundary_batch(kind: str) -> Batch:
    """Crystals with one pair placed within a few fp32 ulps of a cutoff, in
    fp32 Cartesian coordinates (no rounding through fractional coordinates).

    * ``"atom"``: cubic a = 4.3, atoms at (x0, 1, 1) and (x1, 1, 1) with x1
      stepped by single ulps around x0 + 1.7, so the pair through the
      translation (1, 0, 0) is 6 A long (direct distance 1.7 A).
    * ``"bond"``: cubic a = 4.6, x1 around x0 - 1.6, so the pair through
      (1, 0, 0) is 3 A long (direct distance 1.6 A).
    * ``"self"``: one atom at (x0, 1, 1) in a cubic cell whose edge is
      stepped by ulps around 6 A (the atom's own images at the cutoff)."""
    f32 = np.float32
    lat, pos, ptr = [], [], [0]
    for x0 in (0.3, 1.1, 2.189443, 3.0):
        x0 = f32(x0)
        for k in range(-6, 7):
            if kind == "self":
                a = f32(6.0)
                for _ in range(abs(k)):
                    a = np.nextafter(a, f32(np.sign(k) * 10.0))
                lat.append(np.eye(3, dtype=np.float32) * a)
                pos.append(np.array([[x0, 1.0, 1.0]], np.float32))
            else:
                a, off = (f32(4.3), f32(1.7)) if kind == "atom" else (f32(4.6), f32(-1.6))
                x1 = f32(x0 + off)
                for _ in range(abs(k)):
                    x1 = np.nextafter(x1, f32(np.sign(k) * 100.0))
                lat.append(np.eye(3, dtype=np.float32) * a)
                pos.append(np.array([[x0, 1.0, 1.0], [x1, 1.0, 1.0]], np.float32))
            ptr.append(ptr[-1] + len(pos[-1]))
    rng = np.random.default_rng([98, 0, len(kind)])
    P = np.concatenate(pos)
    return Batch(np.asarray(ptr, np.int32), P, np.stack(lat).astype(np.float32),
                 rng.integers(1, N_ELEMENTS + 1, size=len(P)).astype(np.int32))


# --------------------------------------------------------------------------
# Initial weights. The flat layout is the one documented in include/chgnet.h;
# this listing is used only to pick each tensor's initial distribution.
# --------------------------------------------------------------------------

def _param_listing(d: int, T: int, R: int = 31, K: int = 31, magmom: bool = False):
    out = [("W_Z", (N_ELEMENTS, d), "normal"), ("f_a", (R,), "freq"), ("f_b", (R,), "freq"),
           ("W_e", (R, 2 * d), "fan"), ("b_e0", (d,), "fan:%d" % R), ("W_eb", (R, d), "fan"),
           ("W_th", (K, d), "fan"), ("b_th", (d,), "fan:%d" % K)]
    ln = lambda p: [(p + "g_c", (d,), "one"), (p + "b_c", (d,), "zero"), (p + "g_g", (d,), "one"), (p + "b_g", (d,), "zero")]
    for t in range(T):
        out += [("L%d_av_W" % t, (3 * d, 2 * d), "fan"), ("L%d_av_b" % t, (2 * d,), "fan:%d" % (3 * d))]
        out += ln("L%d_av_" % t)
        out += [("L%d_av_Wo" % t, (d, d), "fan"), ("L%d_av_bo" % t, (d,), "fan:%d" % d)]
        out += [("L%d_be_W" % t, (4 * d, 2 * d), "fan"), ("L%d_be_b" % t, (2 * d,), "fan:%d" % (4 * d))]
        out += ln("L%d_be_" % t)
        out += [("L%d_be_Wo" % t, (d, d), "fan"), ("L%d_be_bo" % t, (d,), "fan:%d" % d)]
        if t < T - 1:
            out += [("L%d_an_W" % t, (4 * d, 2 * d), "fan"), ("L%d_an_b" % t, (2 * d,), "fan:%d" % (4 * d))]
            out += ln("L%d_an_" % t)
    for h, o in (("E", 1), ("F", 1), ("S", 9)):
        out += [(h + "_W1", (d, d), "fan"), (h + "_b1", (d,), "fan:%d" % d),
                (h + "_W2", (d, d), "fan"), (h + "_b2", (d,), "fan:%d" % d),
                (h + "_W3", (d, o), "fan"), (h + "_b3", (o,), "fan:%d" % d)]
    if magmom:
        out += [("M_W", (d, 1), "fan"), ("M_b", (1,), "fan:%d" % d)]
    return out


def make_params(d: int, T: int, seed=(0, 1, 0), magmom: bool = False) -> np.ndarray:
    """Flat fp32 parameter vector: U(+-1/sqrt(fan_in)) for weights and biases,
    LayerNorm scale 1 and shift 0, element table N(0,1), frequencies n*pi."""
    rng = np.random.default_rng(list(seed))
    chunks = []
    for _, shape, kind in _param_listing(d, T, magmom=magmom):
        n = int(np.prod(shape))
        if kind == "normal":
            x = rng.standard_normal(n)
        elif kind == "freq":
            x = np.pi * np.arange(1, n + 1)
        elif kind == "one":
            x = np.ones(n)
        elif kind == "zero":
            x = np.zeros(n)
        else:
            fan = shape[0] if kind == "fan" else int(kind.split(":")[1])
            bound = 1.0 / math.sqrt(fan)
            x = rng.uniform(-bound, bound, size=n)
        chunks.append(x)
    return np.concatenate(chunks).astype(np.float32)


def make_targets(batch: Batch, seed=(0, 2, 0), magmom: bool = False):
    """Random targets: per-atom energy N(0,1) per structure, force components
    N(0,1), stress (M + M^T)/2 with M ~ N(0,1); with magmom, also magnetic
    moments |N(0,1)| per atom (drawn after the others)."""
    rng = np.random.default_rng(list(seed))
    S, N = batch.n_struct, batch.n_atoms
    e = rng.standard_normal(S).astype(np.float32)
    f = rng.standard_normal((N, 3)).astype(np.float32)
    m = rng.standard_normal((S, 3, 3))
    s = (0.5 * (m + m.transpose(0, 2, 1))).astype(np.float32)
    if not magmom:
        return e, f, s
    return e, f, s, np.abs(rng.standard_normal(N)).astype(np.float32)


def workload_inputs(name: str, rep: int = 0, magmom: bool = False):
    """(batch, params, targets, d, T) of a named workload."""
    cfg, d, T = WORKLOADS[name]
    batch = make_batch(name, rep)
    params = make_params(d, T, seed=(cfg, 1, rep), magmom=magmom)
    targets = make_targets(batch, seed=(cfg, 2, rep), magmom=magmom)
    return batch, params, targets, d, T
