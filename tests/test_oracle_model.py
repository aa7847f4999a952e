"""Pins of the oracle model: hand-worked GatedMLP, invariances the paper's
heads must satisfy (Eq. (8) rotation equivariance, zero net force of the
pairwise force readout, extensivity, translation and permutation invariance),
finite-difference gradients of the hand-written backward, parameter counts,
the loss and the Adam update."""
import math

import numpy as np
import pytest

from oracle import graph, model
from paper_2412_20796_amd import synth


def _guarded(b, band=2e-3):
    """True if no atom pair lies within `band` of either cutoff."""
    g = graph.build_graph(b.atom_ptr, b.pos, b.lattice, r_atom=6.05, r_bond=3.05)
    d = np.sqrt(g["edge_d2"].astype(np.float64))
    return not (np.any(np.abs(d - 6.0) < band) or np.any(np.abs(d - 3.0) < band))


def _run(hp, b, params):
    g = graph.build_graph(b.atom_ptr, b.pos, b.lattice, hp.r_atom, hp.r_bond)
    E, F, S, _ = model.forward(hp, b, g, params)
    return E, F, S, g


def _small_params(hp, seed, scale=0.3):
    rng = np.random.default_rng(seed)
    n = model.param_count(hp)
    p = rng.standard_normal(n) * scale
    P = model.unpack(hp, p)
    P["f_a"][:] = np.pi * np.arange(1, hp.n_rbf + 1) + 0.05 * rng.standard_normal(hp.n_rbf)
    P["f_b"][:] = np.pi * np.arange(1, hp.n_rbf + 1) + 0.05 * rng.standard_normal(hp.n_rbf)
    return p


def test_param_counts():
    assert model.param_count(model.HParams(d=64, n_layers=4)) == 405_001
    assert model.param_count(model.HParams(d=128, n_layers=5)) == 1_975_753


def test_generator_layout_agrees_with_oracle():
    hp = model.HParams(d=64, n_layers=4)
    P = model.unpack(hp, synth.make_params(64, 4).astype(np.float64))
    np.testing.assert_allclose(P["f_a"], np.pi * np.arange(1, 32), rtol=1e-6)
    np.testing.assert_allclose(P["f_b"], np.pi * np.arange(1, 32), rtol=1e-6)
    for t in range(4):
        assert (P["L%d_av_g_c" % t] == 1).all() and (P["L%d_be_b_g" % t] == 0).all()
    assert "L3_an_W" not in P and "L2_an_W" in P


def test_gated_mlp_hand_worked():
    """d = 2, Fc = identity, gamma = 1, beta = 0. Row 1: z_c = (1, -1) -> LN
    (1, -1)/sqrt(1 + 1e-5); z_g = (0, 0) -> LN (0, 0) -> sigmoid 1/2. Row 2:
    z_c = (3, 3) -> (0, 0), SiLU(0) = 0, so phi = 0. sigmoid(1) =
    0.7310585786300049, hence SiLU(+-1) = 0.7310585786..., -0.2689414213..."""
    P = {"xW": np.eye(4), "xb": np.zeros(4), "xg_c": np.ones(2), "xb_c": np.zeros(2),
         "xg_g": np.ones(2), "xb_g": np.zeros(2)}
    x = np.array([[1.0, -1.0, 0.0, 0.0], [3.0, 3.0, 5.0, -5.0]])
    phi, _ = model.gated_mlp(x, P, "x", 2)
    s = 1.0 / math.sqrt(1.0 + 1e-5)
    sig = lambda y: 1.0 / (1.0 + math.exp(-y))
    assert abs(sig(1.0) - 0.7310585786300049) < 1e-15
    np.testing.assert_allclose(phi[0], [0.5 * s * sig(s), -0.5 * s * sig(-s)], rtol=1e-14)
    np.testing.assert_allclose(phi[1], [0.0, 0.0], atol=1e-15)
    # LN makes phi invariant to a per-row affine map z -> alpha z + c (alpha > 0)
    P2 = dict(P, xW=2.5 * np.eye(4), xb=np.array([1.0, 1.0, -3.0, -3.0]))
    phi2, _ = model.gated_mlp(x, P2, "x", 2)
    np.testing.assert_allclose(phi2, phi, atol=1e-5)  # eps in LN breaks exactness slightly


@pytest.fixture(scope="module")
def small_case():
    hp = model.HParams(d=16, n_layers=3, n_rbf=9, n_fourier=7)
    for seed in range(20):
        b = synth.random_crystals(seed=100 + seed, n_struct=2, n_lo=3, n_hi=6, rho=(0.09, 0.12))
        if _guarded(b):
            g = graph.build_graph(b.atom_ptr, b.pos, b.lattice)
            if len(g["angle_b2"]) > 20:
                return hp, b, _small_params(hp, seed)
    raise RuntimeError("no guarded sample")


def test_net_force_zero_and_rotation(small_case):
    hp, b, p = small_case
    E, F, S, g = _run(hp, b, p)
    for s in range(b.n_struct):
        a0, a1 = b.atom_ptr[s], b.atom_ptr[s + 1]
        assert np.abs(F[a0:a1].sum(0)).max() < 1e-12 * max(1.0, np.abs(F).max())
    rng = np.random.default_rng(0)
    q, _ = np.linalg.qr(rng.standard_normal((3, 3)))
    R = q * np.sign(np.linalg.det(q))
    br = synth.Batch(b.atom_ptr, (b.pos.astype(np.float64) @ R.T).astype(np.float32),
                     (b.lattice.astype(np.float64) @ R.T).astype(np.float32), b.Z)
    E2, F2, S2, g2 = _run(hp, br, p)
    assert len(g2["edge_dst"]) == len(g["edge_dst"])
    np.testing.assert_allclose(E2, E, rtol=1e-5, atol=1e-6)
    np.testing.assert_allclose(F2, F @ R.T, rtol=1e-4, atol=1e-5)
    np.testing.assert_allclose(S2, np.einsum("xa,sab,yb->sxy", R, S, R), rtol=1e-4, atol=1e-5)


def test_translation_permutation_and_lattice_shift(small_case):
    hp, b, p = small_case
    E, F, S, _ = _run(hp, b, p)
    bt = synth.Batch(b.atom_ptr, (b.pos + np.float32(0.37)).astype(np.float32), b.lattice, b.Z)
    E2, F2, S2, _ = _run(hp, bt, p)
    np.testing.assert_allclose(E2, E, rtol=1e-5, atol=1e-6)
    np.testing.assert_allclose(F2, F, rtol=1e-4, atol=1e-5)
    np.testing.assert_allclose(S2, S, rtol=1e-4, atol=1e-5)
    # permute atoms of the first structure
    n0 = b.atom_ptr[1]
    perm = np.concatenate([np.random.default_rng(1).permutation(n0), np.arange(n0, b.n_atoms)])
    bp = synth.Batch(b.atom_ptr, b.pos[perm], b.lattice, b.Z[perm])
    E3, F3, S3, _ = _run(hp, bp, p)
    np.testing.assert_allclose(E3, E, rtol=1e-10)
    np.testing.assert_allclose(F3, F[perm], rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(S3, S, rtol=1e-9, atol=1e-12)
    # move atom 0 by a lattice vector
    pos = b.pos.copy()
    pos[0] = (pos[0].astype(np.float64) + b.lattice[0, 1]).astype(np.float32)
    bs = synth.Batch(b.atom_ptr, pos, b.lattice, b.Z)
    E4, F4, S4, _ = _run(hp, bs, p)
    np.testing.assert_allclose(E4, E, rtol=1e-5, atol=1e-6)
    np.testing.assert_allclose(F4, F, rtol=1e-4, atol=1e-5)


def test_supercell_extensive(small_case):
    hp, b, p = small_case
    L = b.lattice[0].astype(np.float64)
    n = b.atom_ptr[1]
    frac = b.pos[:n].astype(np.float64) @ np.linalg.inv(L)
    b1 = synth.make_custom_batch([L], [frac], [b.Z[:n]])
    L2 = L.copy()
    L2[2] *= 2
    frac2 = np.concatenate([frac * [1, 1, 0.5], (frac + [0, 0, 1]) * [1, 1, 0.5]])
    b2 = synth.make_custom_batch([L2], [frac2], [np.concatenate([b.Z[:n], b.Z[:n]])])
    E1, F1, S1, _ = _run(hp, b1, p)
    E2, F2, S2, _ = _run(hp, b2, p)
    np.testing.assert_allclose(E2, 2 * E1, rtol=1e-5)
    np.testing.assert_allclose(F2, np.concatenate([F1, F1]), rtol=1e-4, atol=1e-5)
    np.testing.assert_allclose(S2, S1, rtol=1e-4, atol=1e-5)


def test_energy_continuous_across_atom_cutoff():
    """e^a carries no bias and the envelope vanishes at 6 A, so an edge that
    appears at the atom-graph cutoff adds nothing to the energy or stress."""
    hp = model.HParams(d=16, n_layers=2, n_rbf=9, n_fourier=7)
    p = _small_params(hp, 7)
    L = np.eye(3) * 20.0
    out = []
    for x in (6.0 - 1e-4, 6.0 + 1e-4):
        frac = np.array([[0.1, 0.1, 0.1], [0.1 + x / 20.0, 0.1, 0.1], [0.1, 0.1 + 2.0 / 20.0, 0.1]])
        b = synth.make_custom_batch([L], [frac], [np.array([3, 8, 26])])
        E, F, S, g = _run(hp, b, p)
        out.append((E, S, len(g["edge_dst"])))
    assert out[0][2] == out[1][2] + 2
    np.testing.assert_allclose(out[0][0], out[1][0], rtol=1e-6, atol=1e-9)
    np.testing.assert_allclose(out[0][1], out[1][1], rtol=1e-6, atol=1e-9)


def _loss(hp, b, g, p, targets):
    E, F, S, cache = model.forward(hp, b, g, p)
    return model.loss_and_grads(E, F, S, cache["g"]["n_per"], *targets)[0]


def test_backward_finite_differences_per_tensor(small_case):
    """Central differences along a random direction restricted to each named
    tensor in turn, against the hand-written backward."""
    hp, b, p = small_case
    g = graph.build_graph(b.atom_ptr, b.pos, b.lattice)
    targets = synth.make_targets(b, seed=(7, 2, 0))
    loss, grad, _, _ = model.step(hp, b, p, targets, graph=g)
    lay, total = model.layout(hp)
    rng = np.random.default_rng(3)
    h = 1e-5
    for name, (off, shape) in lay.items():
        u = np.zeros(total)
        n = int(np.prod(shape))
        u[off:off + n] = rng.standard_normal(n)
        fd = (_loss(hp, b, g, p + h * u, targets) - _loss(hp, b, g, p - h * u, targets)) / (2 * h)
        an = grad @ u
        assert abs(fd - an) <= 1e-6 * max(abs(an), 1e-3), (name, fd, an)


def test_backward_finite_differences_cubic8():
    batch, params, targets, d, T = synth.workload_inputs("cubic8")
    hp = model.HParams(d=d, n_layers=T)
    g = graph.build_graph(batch.atom_ptr, batch.pos, batch.lattice)
    p = params.astype(np.float64)
    loss, grad, _, _ = model.step(hp, batch, p, targets, graph=g)
    rng = np.random.default_rng(5)
    h = 1e-5
    for _ in range(3):
        u = rng.standard_normal(p.shape)
        fd = (_loss(hp, batch, g, p + h * u, targets) - _loss(hp, batch, g, p - h * u, targets)) / (2 * h)
        an = grad @ u
        assert abs(fd - an) <= 1e-6 * abs(an), (fd, an)


def test_loss_hand_values():
    E = np.array([4.0]); n = np.array([2.0]); Et = np.array([1.5])
    F = np.zeros((1, 3)); Ft = np.ones((1, 3))
    S = np.zeros((1, 3, 3)); St = np.eye(3)[None] * 3.0
    loss, dE, dF, dS = model.loss_and_grads(E, F, S, n, Et, Ft, St)
    # 2*(0.5)^2 + 1.5*1 + 0.1*(3*9/9)
    assert abs(loss - (0.5 + 1.5 + 0.3)) < 1e-14
    assert abs(dE[0] - 2 * 2 * 0.5 / 2) < 1e-14
    np.testing.assert_allclose(dF, -1.5 * 2 / 3 * np.ones((1, 3)))
    np.testing.assert_allclose(dS, -0.1 * 2 * 3.0 / 9 * np.eye(3)[None])


def test_adam_first_step_is_signed_lr():
    """With bias correction the first Adam step is -lr * g / (|g| + eps)."""
    p = np.array([1.0, -2.0, 0.5]); g = np.array([0.3, -4.0, 1e-3])
    p1, m, v = model.adam(p, g, np.zeros(3), np.zeros(3), 1e-2, 0.9, 0.999, 1e-8, 1)
    np.testing.assert_allclose(p1, p - 1e-2 * g / (np.abs(g) + 1e-8), rtol=1e-12)
    np.testing.assert_allclose(m, 0.1 * g)
    np.testing.assert_allclose(v, 0.001 * g * g)
