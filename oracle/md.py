"""Oracle: molecular dynamics with the model's direct force head (test
infrastructure; nothing in the GPU library imports it).

The paper times one molecular-dynamics step of single small crystals (Sec. V,
"Molecular dynamics in real applications", Table 2) but does not name the
integrator. Reading: velocity Verlet (Swope, Andersen, Berens and Wilson,
J. Chem. Phys. 76, 637 (1982)) in the NVE ensemble, fixed lattices:

    v <- v + (dt/2) a(x);  x <- x + dt v;  v <- v + (dt/2) a(x)

with a = F / m. Units: positions in Angstrom, time in fs, forces in eV/A,
masses in atomic mass units, so a = F / m * C with C = 1 eV / (A amu)
expressed in A/fs^2 = 1.602176634e-19 / 1e-10 / 1.66053906660e-27 / 1e20
= 0.0096485332157...

Each force evaluation builds the graph anew at the fp32 positions (the cutoff
test is defined on fp32 data) and runs the forward pass of oracle.model.
"""
from __future__ import annotations

import numpy as np

# 1 eV / (Angstrom amu) in Angstrom / fs^2 (CODATA 2018 eV and amu)
ACC = 1.602176634e-19 / 1e-10 / 1.66053906660e-27 / 1e20


def velocity_verlet(x, v, inv_mass, dt, n_steps, force_fn, f=None):
    """n_steps of velocity Verlet from (x, v); force_fn(x) -> forces [N,3].
    Returns (x, v, f) with f the forces at the final positions."""
    x = np.asarray(x, dtype=np.float64).copy()
    v = np.asarray(v, dtype=np.float64).copy()
    im = ACC * np.asarray(inv_mass, dtype=np.float64)[:, None]
    f = force_fn(x) if f is None else np.asarray(f, dtype=np.float64)
    for _ in range(n_steps):
        v = v + 0.5 * dt * im * f
        x = x + dt * v
        f = force_fn(x)
        v = v + 0.5 * dt * im * f
    return x, v, f


def model_force_fn(hp, batch, params, record=None):
    """force_fn for velocity_verlet: the model's forces at positions x (the
    batch's lattices and species); `record` collects (energy, stress, graph)
    of every evaluation when given."""
    from . import graph as og
    from . import model as om

    p = np.asarray(params, dtype=np.float64)

    def fn(x):
        pos = np.asarray(x, dtype=np.float64).astype(np.float32)
        b = type(batch)(batch.atom_ptr, pos, batch.lattice, batch.Z)
        g = og.build_graph(b.atom_ptr, b.pos, b.lattice, hp.r_atom, hp.r_bond)
        E, F, S, _ = om.forward(hp, b, g, p)
        if record is not None:
            record.append((E, S, g))
        return F

    return fn
