"""Pins of the oracle's conservative readout (F = -dE/dr, sigma = (1/V)
dE/d(eps)): the basis derivatives against central differences and the
factored envelope derivative; forces and stresses against central
differences of the energy in the positions and in a homogeneous strain of
positions and lattice (graph held fixed, fp64 positions); zero net force,
rotation equivariance and symmetry of the stress; a collinear bond pair."""
import math

import numpy as np
import pytest

from oracle import graph, model
from paper_2412_20796_amd import synth

from test_oracle_model import _guarded, _small_params


def test_basis_derivatives():
    p, c = 8, 6.0
    x = np.linspace(0.05, 0.999, 37)
    np.testing.assert_allclose(model.envelope_dx(x, p), -p * (p + 1) * (p + 2) / 2 * x ** (p - 1) * (1 - x) ** 2,
                               rtol=1e-9, atol=1e-12)
    r = np.linspace(0.7, 5.99, 41)
    f = math.pi * np.arange(1, 32) + 0.1
    h = 1e-6
    fd = (model.srbf(r + h, f, c, p) - model.srbf(r - h, f, c, p)) / (2 * h)
    np.testing.assert_allclose(model.srbf_dr(r, f, c, p), fd, rtol=1e-6, atol=1e-7)
    th = np.linspace(0.01, math.pi - 0.01, 29)
    fd = (model.fourier(th + h, 31) - model.fourier(th - h, 31)) / (2 * h)
    np.testing.assert_allclose(model.fourier_dtheta(th, 31), fd, rtol=1e-6, atol=1e-7)


@pytest.fixture(scope="module")
def case():
    for seed in range(20):
        b = synth.random_crystals(seed=100 + seed, n_struct=2, n_lo=3, n_hi=6, rho=(0.09, 0.12))
        if _guarded(b):
            g = graph.build_graph(b.atom_ptr, b.pos, b.lattice)
            if len(g["angle_b2"]) > 20:
                return b, g, seed
    raise RuntimeError("no guarded sample")


def _energy(hp, b, g, p, pos, lat):
    bb = synth.Batch(b.atom_ptr, pos, lat, b.Z)
    return model.forward(model.HParams(**{**hp.__dict__, "conservative": False}), bb, g, p)[0]


@pytest.mark.parametrize("sequential", [False, True])
def test_forces_and_stress_are_energy_derivatives(case, sequential):
    b, g, seed = case
    hp = model.HParams(d=16, n_layers=3, n_rbf=9, n_fourier=7, conservative=True, sequential=sequential)
    p = _small_params(hp, seed)
    E, F, S, _ = model.forward(hp, b, g, p)
    pos = b.pos.astype(np.float64)
    lat = b.lattice.astype(np.float64)
    h = 1e-5
    for i in range(b.n_atoms):
        for c in range(3):
            dp = np.zeros_like(pos)
            dp[i, c] = h
            s = np.searchsorted(b.atom_ptr, i, side="right") - 1
            fd = (_energy(hp, b, g, p, pos + dp, lat)[s] - _energy(hp, b, g, p, pos - dp, lat)[s]) / (2 * h)
            assert abs(-fd - F[i, c]) <= 1e-6 * max(1.0, abs(F[i, c])), (i, c, -fd, F[i, c])
    vol = np.abs(np.linalg.det(lat))
    for a in range(3):
        for c in range(3):
            eps = np.zeros((3, 3))
            eps[a, c] = h
            up = _energy(hp, b, g, p, pos @ (np.eye(3) + eps).T, lat @ (np.eye(3) + eps).T)
            dn = _energy(hp, b, g, p, pos @ (np.eye(3) - eps).T, lat @ (np.eye(3) - eps).T)
            fd = (up - dn) / (2 * h) / vol
            np.testing.assert_allclose(S[:, a, c], fd, rtol=1e-6, atol=1e-8)


def test_conservative_invariances(case):
    b, g, seed = case
    hp = model.HParams(d=16, n_layers=3, n_rbf=9, n_fourier=7, conservative=True)
    p = _small_params(hp, seed)
    E, F, S, _ = model.forward(hp, b, g, p)
    for s in range(b.n_struct):
        a0, a1 = b.atom_ptr[s], b.atom_ptr[s + 1]
        assert np.abs(F[a0:a1].sum(0)).max() < 1e-10 * max(1.0, np.abs(F).max())
    np.testing.assert_allclose(S, S.transpose(0, 2, 1), rtol=1e-9, atol=1e-12)
    rng = np.random.default_rng(0)
    q, _ = np.linalg.qr(rng.standard_normal((3, 3)))
    R = q * np.sign(np.linalg.det(q))
    br = synth.Batch(b.atom_ptr, b.pos.astype(np.float64) @ R.T, b.lattice.astype(np.float64) @ R.T, b.Z)
    E2, F2, S2, _ = model.forward(hp, br, g, p)
    np.testing.assert_allclose(E2, E, rtol=1e-10)
    np.testing.assert_allclose(F2, F @ R.T, rtol=1e-8, atol=1e-10)
    np.testing.assert_allclose(S2, np.einsum("xa,sab,yb->sxy", R, S, R), rtol=1e-8, atol=1e-10)


def test_collinear_bond_pair():
    """Three atoms on a line 2 A apart in a 20 A cell: the middle atom's two
    bonds are exactly antiparallel (theta = pi). The readout stays finite and
    its component along the line matches the energy's central difference."""
    hp = model.HParams(d=16, n_layers=2, n_rbf=9, n_fourier=7, conservative=True)
    p = _small_params(hp, 4)
    L = np.eye(3) * 20.0
    frac = np.array([[0.3, 0.5, 0.5], [0.4, 0.5, 0.5], [0.5, 0.5, 0.5]])
    b = synth.make_custom_batch([L], [frac], [np.array([8, 26, 8])])
    g = graph.build_graph(b.atom_ptr, b.pos, b.lattice)
    E, F, S, cache = model.forward(hp, b, g, p)
    assert np.isclose(cache["g"]["theta"], math.pi).any()
    assert np.isfinite(F).all() and np.isfinite(S).all()
    pos = b.pos.astype(np.float64)
    h = 1e-5
    for i in range(3):
        dp = np.zeros_like(pos)
        dp[i, 0] = h
        fd = (_energy(hp, b, g, p, pos + dp, b.lattice)[0] - _energy(hp, b, g, p, pos - dp, b.lattice)[0]) / (2 * h)
        assert abs(-fd - F[i, 0]) <= 1e-6 * max(1.0, abs(F[i, 0]))


def test_conservative_training_step_refused(case):
    b, g, seed = case
    hp = model.HParams(d=16, n_layers=2, n_rbf=9, n_fourier=7, conservative=True)
    with pytest.raises(NotImplementedError):
        model.step(hp, b, _small_params(hp, 0), synth.make_targets(b), graph=g)


def test_md_energy_conservation_is_second_order():
    """With F = -dE/dr, velocity Verlet conserves E + kinetic energy up to an
    O(dt^2) error: halving dt cuts the largest deviation over the same
    trajectory time by about 4. The graph is held fixed and positions stay in
    fp64, so E is a smooth function of the positions."""
    from oracle import md

    hp = model.HParams(d=16, n_layers=2, n_rbf=9, n_fourier=7, conservative=True)
    b = synth.make_batch("cubic8")
    g0 = graph.build_graph(b.atom_ptr, b.pos, b.lattice)
    p = _small_params(hp, 2, scale=0.3)
    rng = np.random.default_rng(5)
    v0 = rng.standard_normal((b.n_atoms, 3)) * 0.05
    mass = rng.uniform(20.0, 60.0, b.n_atoms)

    def run(dt, n):
        energies = []

        def fn(x):
            E, F, _, _ = model.forward(hp, synth.Batch(b.atom_ptr, x, b.lattice, b.Z), g0, p)
            energies.append(E.sum())
            return F

        x, v, f = b.pos.astype(np.float64), v0.copy(), None
        tot = []
        for _ in range(n):
            x, v, f = md.velocity_verlet(x, v, 1.0 / mass, dt, 1, fn, f=f)
            tot.append(energies[-1] + 0.5 * (mass[:, None] * v * v).sum() / md.ACC)
        return np.abs(np.array(tot) - tot[0]).max()

    e1, e2, e3 = run(1.0, 8), run(0.5, 16), run(0.25, 32)
    assert e1 > 1e-6
    # an inconsistent force (F != -grad E) leaves an O(dt) or O(1) drift: ratios 2 or 1
    assert 3.5 < e1 / e2 < 5.0 and 3.5 < e2 / e3 < 5.0, (e1, e2, e3)
