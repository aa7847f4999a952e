"""Pins of the oracle's model variants: the Huber loss (Sec. IV), the
magnetic-moment head and the sequential interaction block of Eq. (10).

Huber values are worked by hand; the large-threshold limit is half the squared
error; the moments are rotation, translation and permutation invariant and
non-negative; the Eq. (10) block keeps the invariances of Eq. (8), reduces to
the Eq. (11) block when the atom and bond updates vanish, and the hand-written
backward of every variant agrees with central differences."""
import numpy as np
import pytest

from oracle import graph, model
from paper_2412_20796_amd import synth

from test_oracle_model import _guarded, _small_params


def test_huber_hand_values():
    # delta = 0.1: |0.05| <= delta -> 0.05^2 / 2; |-0.3| > delta -> 0.1 (0.3 - 0.05)
    h, dh = model.huber(np.array([0.05, -0.3, 0.1, 0.0]), 0.1)
    np.testing.assert_allclose(h, [0.00125, 0.025, 0.005, 0.0], rtol=1e-14, atol=1e-18)
    np.testing.assert_allclose(dh, [0.05, -0.1, 0.1, 0.0], rtol=1e-14)


def test_huber_loss_hand_values():
    E = np.array([4.0]); n = np.array([2.0]); Et = np.array([1.5])  # r = 0.5
    F = np.array([[0.0, 0.02, -1.0]]); Ft = np.zeros((1, 3))
    S = np.zeros((1, 3, 3)); St = np.zeros((1, 3, 3)); St[0, 1, 2] = -0.04
    loss, dE, dF, dS = model.loss_and_grads(E, F, S, n, Et, Ft, St, delta=0.1)
    le = 0.1 * (0.5 - 0.05)
    lf = (0.5 * 0.02 ** 2 + 0.1 * (1.0 - 0.05)) / 3
    ls = 0.5 * 0.04 ** 2 / 9
    assert abs(loss - (2 * le + 1.5 * lf + 0.1 * ls)) < 1e-15
    assert abs(dE[0] - 2 * 0.1 / 2) < 1e-15
    np.testing.assert_allclose(dF, 1.5 / 3 * np.array([[0.0, 0.02, -0.1]]), rtol=1e-14)
    expect = np.zeros((1, 3, 3)); expect[0, 1, 2] = 0.1 * 0.04 / 9
    np.testing.assert_allclose(dS, expect, rtol=1e-14, atol=1e-18)


def test_huber_large_threshold_is_half_squared_error():
    rng = np.random.default_rng(0)
    S, N = 3, 7
    args = (rng.standard_normal(S), rng.standard_normal((N, 3)), rng.standard_normal((S, 3, 3)),
            np.array([2.0, 3.0, 2.0]), rng.standard_normal(S), rng.standard_normal((N, 3)),
            rng.standard_normal((S, 3, 3)))
    mse = model.loss_and_grads(*args)
    hub = model.loss_and_grads(*args, delta=1e9)
    for a, b in zip(mse, hub):
        np.testing.assert_allclose(b, 0.5 * np.asarray(a), rtol=1e-14)
    m = np.abs(rng.standard_normal(N)); mt = np.abs(rng.standard_normal(N))
    l2, g2 = model.magmom_loss(m, mt, 0.1)
    assert abs(l2 - 0.1 * np.mean((m - mt) ** 2)) < 1e-15
    np.testing.assert_allclose(g2, 0.1 * 2 * (m - mt) / N, rtol=1e-14)
    lh, gh = model.magmom_loss(m, mt, 0.1, delta=1e9)
    assert abs(lh - 0.5 * l2) < 1e-15
    np.testing.assert_allclose(gh, 0.5 * g2, rtol=1e-14)


@pytest.fixture(scope="module")
def case():
    for seed in range(20):
        b = synth.random_crystals(seed=100 + seed, n_struct=2, n_lo=3, n_hi=6, rho=(0.09, 0.12))
        if _guarded(b):
            g = graph.build_graph(b.atom_ptr, b.pos, b.lattice)
            if len(g["angle_b2"]) > 20:
                return b, seed
    raise RuntimeError("no guarded sample")


def _hp(**kw):
    return model.HParams(d=16, n_layers=3, n_rbf=9, n_fourier=7, **kw)


def _run(hp, b, p):
    g = graph.build_graph(b.atom_ptr, b.pos, b.lattice, hp.r_atom, hp.r_bond)
    E, F, S, cache = model.forward(hp, b, g, p)
    return E, F, S, cache["magmom"]


def test_magmom_layout_appends_head():
    base = model.layout(_hp())[1]
    lay, total = model.layout(_hp(magmom=True))
    assert total == base + 16 + 1 and lay["M_W"] == (base, (16, 1)) and lay["M_b"] == (base + 16, (1,))
    # the generator appends the same two tensors last
    p0 = synth.make_params(64, 4, seed=(1, 1, 0))
    p1 = synth.make_params(64, 4, seed=(1, 1, 0), magmom=True)
    assert p1.shape[0] == model.param_count(model.HParams(magmom=True)) == 405_001 + 65
    np.testing.assert_array_equal(p1[:p0.shape[0]], p0)


def test_magmom_invariances(case):
    b, seed = case
    hp = _hp(magmom=True)
    p = _small_params(hp, seed)
    E, F, S, M = _run(hp, b, p)
    assert M.shape == (b.n_atoms,) and (M >= 0).all() and M.max() > 0
    # energies, forces and stress do not depend on the extra head
    hp0 = _hp()
    E0, F0, S0, M0 = _run(hp0, b, p[:model.param_count(hp0)])
    assert M0 is None
    np.testing.assert_array_equal(E0, E)
    np.testing.assert_array_equal(F0, F)
    rng = np.random.default_rng(0)
    q, _ = np.linalg.qr(rng.standard_normal((3, 3)))
    R = q * np.sign(np.linalg.det(q))
    br = synth.Batch(b.atom_ptr, (b.pos.astype(np.float64) @ R.T).astype(np.float32),
                     (b.lattice.astype(np.float64) @ R.T).astype(np.float32), b.Z)
    np.testing.assert_allclose(_run(hp, br, p)[3], M, rtol=1e-5, atol=1e-7)
    n0 = b.atom_ptr[1]
    perm = np.concatenate([np.random.default_rng(1).permutation(n0), np.arange(n0, b.n_atoms)])
    bp = synth.Batch(b.atom_ptr, b.pos[perm], b.lattice, b.Z[perm])
    np.testing.assert_allclose(_run(hp, bp, p)[3], M[perm], rtol=1e-10)
    # w_m = 0: every moment is |b_m|
    P = model.unpack(hp, p.copy())
    P["M_W"][:] = 0.0
    P["M_b"][:] = -0.7
    flat = np.concatenate([P[k].reshape(-1) for k in model.layout(hp)[0]])
    np.testing.assert_allclose(_run(hp, b, flat)[3], 0.7, rtol=1e-15)


def test_sequential_invariances(case):
    b, seed = case
    hp = _hp(sequential=True)
    p = _small_params(hp, seed)
    E, F, S, _ = _run(hp, b, p)
    for s in range(b.n_struct):
        a0, a1 = b.atom_ptr[s], b.atom_ptr[s + 1]
        assert np.abs(F[a0:a1].sum(0)).max() < 1e-12 * max(1.0, np.abs(F).max())
    rng = np.random.default_rng(2)
    q, _ = np.linalg.qr(rng.standard_normal((3, 3)))
    R = q * np.sign(np.linalg.det(q))
    br = synth.Batch(b.atom_ptr, (b.pos.astype(np.float64) @ R.T).astype(np.float32),
                     (b.lattice.astype(np.float64) @ R.T).astype(np.float32), b.Z)
    E2, F2, S2, _ = _run(hp, br, p)
    np.testing.assert_allclose(E2, E, rtol=1e-5, atol=1e-6)
    np.testing.assert_allclose(F2, F @ R.T, rtol=1e-4, atol=1e-5)
    np.testing.assert_allclose(S2, np.einsum("xa,sab,yb->sxy", R, S, R), rtol=1e-4, atol=1e-5)
    # the two block orders give different models
    E11, F11, S11, _ = _run(_hp(), b, p)
    assert np.abs(F11 - F).max() > 1e-3 * np.abs(F).max()


def test_sequential_reduces_to_parallel_without_updates(case):
    """With zero output linears of the atom and bond updates, v^{t+1} = v^t and
    e^{t+1} = e^t, so Eq. (10) and Eq. (11) read the same inputs."""
    b, seed = case
    hp = _hp(sequential=True)
    P = model.unpack(hp, _small_params(hp, seed))
    for t in range(hp.n_layers):
        for k in ("av_Wo", "av_bo", "be_Wo", "be_bo"):
            P["L%d_%s" % (t, k)][:] = 0.0
    flat = np.concatenate([P[k].reshape(-1) for k in model.layout(hp)[0]])
    out_seq = _run(hp, b, flat)
    out_par = _run(_hp(), b, flat)
    for x, y in zip(out_seq[:3], out_par[:3]):
        np.testing.assert_array_equal(x, y)


def _loss(hp, b, g, p, targets, delta):
    E, F, S, cache = model.forward(hp, b, g, p)
    loss = model.loss_and_grads(E, F, S, cache["g"]["n_per"], *targets[:3], delta=delta)[0]
    if hp.magmom:
        loss += model.magmom_loss(cache["magmom"], targets[3], 0.1, delta)[0]
    return loss


@pytest.mark.parametrize("variant", [dict(magmom=True), dict(sequential=True), dict(magmom=True, sequential=True)])
@pytest.mark.parametrize("delta", [None, 0.1])
def test_variant_backward_finite_differences(case, variant, delta):
    """Central differences along a random direction restricted to each named
    tensor, against the hand-written backward."""
    b, seed = case
    hp = _hp(**variant)
    p = _small_params(hp, seed)
    g = graph.build_graph(b.atom_ptr, b.pos, b.lattice)
    targets = synth.make_targets(b, seed=(7, 2, 0), magmom=hp.magmom)
    loss, grad, _, _ = model.step(hp, b, p, targets, graph=g, delta=delta)
    assert abs(loss - _loss(hp, b, g, p, targets, delta)) <= 1e-14 * abs(loss)
    lay, total = model.layout(hp)
    rng = np.random.default_rng(3)
    h = 1e-5
    for name, (off, shape) in lay.items():
        u = np.zeros(total)
        n = int(np.prod(shape))
        u[off:off + n] = rng.standard_normal(n)
        fd = (_loss(hp, b, g, p + h * u, targets, delta) - _loss(hp, b, g, p - h * u, targets, delta)) / (2 * h)
        an = grad @ u
        assert abs(fd - an) <= 1e-6 * max(abs(an), 1e-3), (name, fd, an)
