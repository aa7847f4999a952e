"""Pins of the autodiff oracle (an independent PyTorch fp64 transcription of
the forward, differentiated by autograd) and, through it, of the training
gradient through the conservative readout, which needs second derivatives:

* its forward equals oracle.model's (direct heads; Eq. (11) and Eq. (10);
  magnetic-moment head);
* its loss gradient equals oracle.model's hand-written backward (squared and
  Huber errors, magnetic moments): a second, independent derivation;
* its conservative F = -dE/dr and sigma = (1/V) dE/d(eps) equal
  oracle.model's conservative readout (itself pinned to central
  differences of the energy);
* the weight gradient of the loss through the conservative readout equals
  central differences of oracle.model's conservative loss along random
  directions in parameter space."""
import numpy as np
import pytest

from oracle import autodiff, graph, model
from paper_2412_20796_amd import synth

from test_oracle_model import _guarded, _small_params


@pytest.fixture(scope="module")
def case():
    for seed in range(30):
        b = synth.random_crystals(seed=300 + seed, n_struct=2, n_lo=3, n_hi=6, rho=(0.09, 0.12))
        if _guarded(b):
            g = graph.build_graph(b.atom_ptr, b.pos, b.lattice)
            if len(g["angle_b2"]) > 20:
                return b, g, seed
    raise RuntimeError("no guarded sample")


def _hp(**kw):
    return model.HParams(d=16, n_layers=3, n_rbf=9, n_fourier=7, **kw)


def _np_loss(hp, b, g, p, targets, delta, w_m=0.1):
    E, F, S, cache = model.forward(hp, b, g, p)
    loss, dE, dF, dS = model.loss_and_grads(E, F, S, cache["g"]["n_per"], *targets[:3], delta=delta)
    dM = None
    if hp.magmom:
        lm, dM = model.magmom_loss(cache["magmom"], targets[3], w_m, delta)
        loss += lm
    return loss, (cache, dE, dF, dS, dM)


@pytest.mark.parametrize("kw", [{}, {"sequential": True}, {"magmom": True}])
def test_forward_matches(case, kw):
    b, g, seed = case
    hp = _hp(**kw)
    p = _small_params(hp, seed)
    E, F, S, cache = model.forward(hp, b, g, p)
    tE, tF, tS, tM = autodiff.numpy_outputs(hp, b, g, p)
    np.testing.assert_allclose(tE, E, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(tF, F, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(tS, S, rtol=1e-10, atol=1e-12)
    if hp.magmom:
        np.testing.assert_allclose(tM, cache["magmom"], rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("kw,delta", [({}, None), ({"sequential": True}, None), ({}, 0.5), ({"magmom": True}, 0.3)])
def test_hand_backward_matches_autograd(case, kw, delta):
    b, g, seed = case
    hp = _hp(**kw)
    p = _small_params(hp, seed)
    targets = synth.make_targets(b, seed=(7, 2, seed), magmom=hp.magmom)
    loss, (cache, dE, dF, dS, dM) = _np_loss(hp, b, g, p, targets, delta)
    grad = model.backward(hp, cache, dE, dF, dS, dM)
    tl, tg = autodiff.loss_and_grad(hp, b, g, p, targets, delta=delta)
    assert abs(tl - loss) <= 1e-11 * abs(loss)
    np.testing.assert_allclose(tg, grad, rtol=1e-8, atol=1e-10 * np.abs(grad).max())


@pytest.mark.parametrize("kw", [{}, {"sequential": True}])
def test_conservative_readout_matches(case, kw):
    b, g, seed = case
    hp = _hp(conservative=True, **kw)
    p = _small_params(hp, seed)
    E, F, S, _ = model.forward(hp, b, g, p)
    tE, tF, tS, _ = autodiff.numpy_outputs(hp, b, g, p)
    np.testing.assert_allclose(tE, E, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(tF, F, rtol=1e-9, atol=1e-11 * np.abs(F).max())
    np.testing.assert_allclose(tS, S, rtol=1e-9, atol=1e-11 * np.abs(S).max())


@pytest.mark.parametrize("kw,delta", [({}, None), ({"sequential": True}, None), ({}, 0.4)])
def test_conservative_training_gradient_fd(case, kw, delta):
    """d loss / d theta through F = -dE/dr against central differences of
    the hand-derived conservative loss (three random unit directions)."""
    b, g, seed = case
    hp = _hp(conservative=True, **kw)
    p = _small_params(hp, seed)
    targets = synth.make_targets(b, seed=(7, 2, 40 + seed))
    loss, tg = autodiff.loss_and_grad(hp, b, g, p, targets, delta=delta)
    assert abs(loss - _np_loss(hp, b, g, p, targets, delta)[0]) <= 1e-10 * abs(loss)
    rng = np.random.default_rng(seed)
    h = 1e-5
    for _ in range(3):
        u = rng.standard_normal(p.shape)
        u /= np.linalg.norm(u)
        fd = (_np_loss(hp, b, g, p + h * u, targets, delta)[0] - _np_loss(hp, b, g, p - h * u, targets, delta)[0]) / (2 * h)
        assert abs(float(tg @ u) - fd) <= 1e-6 * max(abs(fd), 1e-3 * np.linalg.norm(tg)), (float(tg @ u), fd)


def test_conservative_gradient_differs_from_direct_heads(case):
    """With the conservative readout the force and stress heads are unused:
    their weights get no gradient, while every interaction weight does."""
    b, g, seed = case
    hp = _hp(conservative=True)
    p = _small_params(hp, seed)
    _, tg = autodiff.loss_and_grad(hp, b, g, p, synth.make_targets(b, seed=(7, 2, seed)))
    lay, _ = model.layout(hp)
    for name, (o, s) in lay.items():
        n = int(np.prod(s))
        if name.startswith(("F_", "S_")):
            assert np.all(tg[o:o + n] == 0.0), name
    o, s = lay["L0_av_W"]
    assert np.abs(tg[o:o + int(np.prod(s))]).max() > 0


@pytest.mark.parametrize("delta", [None, 0.4])
def test_loss_gradient_is_the_tangent_of_the_weight_gradient(case, delta):
    """The identity behind the forward-over-reverse GPU path: with the loss
    gradients l_E, l_F, l_sigma of the outputs, the loss gradient through the
    conservative readout equals d/dh at h = 0 of the first-order weight
    gradient of sum_s (1 + h l_E,s) E_s at positions r - h l_F and strain
    h l_sigma / V (central differences in h, fp64)."""
    import torch

    b, g, seed = case
    hp = _hp(conservative=True)
    p = _small_params(hp, seed)
    targets = synth.make_targets(b, seed=(7, 2, 80 + seed))
    _, tg = autodiff.loss_and_grad(hp, b, g, p, targets, delta=delta)
    ix = autodiff._indices(b, g)
    E, F, S, _, _ = autodiff.outputs(hp, b, g, p, create_graph=False, ix=ix)
    E, F, S = (x.detach().requires_grad_(True) for x in (E, F, S))
    Et, Ft, St = (torch.as_tensor(x, dtype=torch.float64) for x in targets[:3])
    n = torch.as_tensor(ix["n_per"])
    pw = lambda r: r * r if delta is None else torch.where(r.abs() <= delta, 0.5 * r * r, delta * (r.abs() - 0.5 * delta))
    loss = 2.0 * pw(E / n - Et).mean() + 1.5 * pw(F - Ft).mean() + 0.1 * pw(S - St).mean()
    lE, lF, lS = torch.autograd.grad(loss, (E, F, S))
    vol = torch.abs(torch.linalg.det(torch.as_tensor(b.lattice, dtype=torch.float64)))
    pos0 = torch.as_tensor(b.pos, dtype=torch.float64)

    def weight_grad(h):
        pt = torch.tensor(p, dtype=torch.float64, requires_grad=True)
        En, _, _, _ = autodiff.forward(hp, b, g, pt, pos=pos0 - h * lF, strain=h * lS / vol[:, None, None], ix=ix)
        (gr,) = torch.autograd.grad(((1.0 + h * lE) * En).sum(), pt)
        return gr.numpy()

    h = 1e-5
    tangent = (weight_grad(h) - weight_grad(-h)) / (2 * h)
    np.testing.assert_allclose(tangent, tg, rtol=1e-5, atol=1e-7 * np.abs(tg).max())
