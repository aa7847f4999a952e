"""Pins of the molecular-dynamics oracle: velocity Verlet against the closed
forms of free motion and of a harmonic oscillator, the unit constant, time
reversibility with the model's forces, and conservation of each crystal's
momentum (the symmetrised force head gives zero net force)."""
import math

import numpy as np

from oracle import md, model
from paper_2412_20796_amd import synth


def test_unit_constant():
    """Independently through the Faraday constant: e/u = F / M_u with
    F = e N_A = 96485.33212 C/mol and M_u = 0.99999999965e-3 kg/mol (CODATA
    2018); a force of 1 eV/A on 1 u accelerates by (e/u) * 1e10 m/s^2, which is
    (e/u) * 1e-10 A/fs^2."""
    assert abs(md.ACC / (96485.33212 / 0.99999999965e-3 * 1e-10) - 1.0) < 1e-9


def test_free_motion():
    rng = np.random.default_rng(0)
    x0, v0 = rng.standard_normal((5, 3)), rng.standard_normal((5, 3))
    x, v, f = md.velocity_verlet(x0, v0, np.ones(5), 0.5, 7, lambda x: np.zeros_like(x))
    np.testing.assert_allclose(x, x0 + 3.5 * v0, rtol=1e-14, atol=1e-14)
    np.testing.assert_array_equal(v, v0)


def test_harmonic_closed_form():
    """F = -k x. Velocity Verlet maps (x_n, x_{n-1}) like the central
    difference x_{n+1} = 2 x_n - x_{n-1} - (w dt)^2 x_n, whose solution is
    x_n = A cos(n phi) + B sin(n phi) with cos(phi) = 1 - (w dt)^2 / 2; its
    half-step velocities give v_n = (x_{n+1} - x_{n-1}) / (2 dt)."""
    k, m, dt, n = 2.0, 3.0, 0.7, 25
    w2 = k * md.ACC / m
    x0, v0 = np.array([[0.3, -1.2, 0.0]]), np.array([[0.05, 0.0, -0.02]])
    x, v, f = md.velocity_verlet(x0, v0, np.array([1.0 / m]), dt, n, lambda x: -k * x)
    phi = math.acos(1.0 - 0.5 * w2 * dt * dt)
    x1 = x0 + dt * v0 - 0.5 * dt * dt * w2 * x0
    B = (x1 - x0 * math.cos(phi)) / math.sin(phi)

    def xn(j):
        return x0 * math.cos(j * phi) + B * math.sin(j * phi)

    np.testing.assert_allclose(x, xn(n), rtol=1e-10, atol=1e-13)
    np.testing.assert_allclose(v, (xn(n + 1) - xn(n - 1)) / (2 * dt), rtol=1e-9, atol=1e-13)
    np.testing.assert_allclose(f, -k * x, rtol=1e-15)


def _case():
    b = synth.make_batch("cubic8")
    hp = model.HParams(d=16, n_layers=2, n_rbf=9, n_fourier=7)
    rng = np.random.default_rng(1)
    p = rng.standard_normal(model.param_count(hp)) * 0.3
    P = model.unpack(hp, p)
    P["f_a"][:] = np.pi * np.arange(1, 10)
    P["f_b"][:] = np.pi * np.arange(1, 10)
    v0 = rng.standard_normal((b.n_atoms, 3)) * 0.02
    inv_m = 1.0 / rng.uniform(6.0, 60.0, b.n_atoms)
    return hp, b, p, v0, inv_m


def test_time_reversible_with_model_forces():
    hp, b, p, v0, inv_m = _case()
    fn = md.model_force_fn(hp, b, p)
    x0 = b.pos.astype(np.float64)
    x, v, f = md.velocity_verlet(x0, v0, inv_m, 1.0, 4, fn)
    assert np.abs(x - x0).max() > 1e-3
    xb, vb, _ = md.velocity_verlet(x, -v, inv_m, 1.0, 4, fn, f=f)
    np.testing.assert_allclose(xb, x0, rtol=0, atol=1e-11)
    np.testing.assert_allclose(-vb, v0, rtol=0, atol=1e-12)


def test_momentum_conserved():
    hp, b, p, v0, inv_m = _case()
    rec = []
    x, v, f = md.velocity_verlet(b.pos, v0, inv_m, 1.0, 3, md.model_force_fn(hp, b, p, rec))
    assert len(rec) == 4
    mass = 1.0 / inv_m[:, None]
    np.testing.assert_allclose((mass * v).sum(0), (mass * v0).sum(0), rtol=0, atol=1e-11)
