"""GPU weight gradient through the conservative readout (F = -dE/dr, sigma =
(1/V) dE/d(eps); the library runs the forward pass and the weight backward in
dual numbers) against the fp64 autodiff oracle, which differentiates the loss
through autograd's own dE/dr and dE/d(eps) (second derivatives by
create_graph): the training step's loss and gradient (squared and Huber
errors) and chgnet_backward with random output gradients, on the cubic8
workload, random small batches, the magnetic-moment head (its loss term
is first order) and sparse cells (no bonds, no angles, no edges); at the
full triclinic40 (d = 64, T = 4) and wide128 (d = 128, T = 5) sizes, output
gradients on a sample of structures against the oracle on those structures
alone (crystals of a batch are independent and the gradient is linear in
the output gradients); the reference block of Eq. (10) on cubic8, random
batches, the moment head and d = 128, and through chgnet_backward.

Tolerance per parameter tensor: |gpu - ref| <= 3e-5 m + 1e-4 |ref|, with m
the larger of the tensor's max|ref| and 1e-2 of the whole gradient's (a
tensor whose exact gradient vanishes, such as the energy bias when the
energy errors of a batch cancel, is held to rounding of the whole sum).
The relative term is the first-order tests' 1e-4. The fp32 path forms each
gradient term as a product of a first derivative (as accurate as the
direct-head gradients, about 1e-5 relative) with tangents that pass through
the same chain once more, and sums terms of both signs over every edge and
angle, so its absolute error scales with the tensor's largest entry rather
than with each entry: measured at most 5e-6 of m on every tensor but one,
and 1.8e-5 of m on the energy bias of a batch whose energy errors cancel."""
import numpy as np
import pytest

from oracle import autodiff
from oracle import graph as og
from oracle import model as om
from paper_2412_20796_amd import synth

pytestmark = pytest.mark.gpu

ATOL_REL, RTOL = 3e-5, 1e-4


@pytest.fixture(scope="module")
def bd():
    import torch

    from paper_2412_20796_amd import binding

    assert torch.cuda.is_available()
    binding.lib()
    return binding


def _dev(x):
    import torch

    return torch.as_tensor(np.ascontiguousarray(x)).to("cuda")


def _assert_grad(got, ref, ohp, what):
    lay, _ = om.layout(ohp)
    gscale = np.abs(ref).max()
    worst = []
    for name, (o, s) in lay.items():
        n = int(np.prod(s))
        g, r = got[o:o + n].astype(np.float64), ref[o:o + n]
        scale = max(np.abs(r).max(), 1e-2 * gscale)
        err = np.abs(g - r)
        bad = err > ATOL_REL * scale + RTOL * np.abs(r)
        worst.append((float(err.max() / max(scale, 1e-30)), name))
        if bad.any():
            k = int(np.argmax(err - ATOL_REL * scale - RTOL * np.abs(r)))
            raise AssertionError("%s grad %s: %d/%d outside tolerance; worst at %d: gpu %.9g ref %.9g (max|ref| %.3g)"
                                 % (what, name, int(bad.sum()), n, k, g[k], r[k], scale))
    worst.sort(reverse=True)
    print(what, "largest error / max|ref|:", ", ".join("%s %.2e" % (nm, e) for e, nm in worst[:3]), flush=True)


def _setup(bd, b, d, T, **kw):
    hp = bd.hparams(d=d, n_layers=T, conservative=True, **kw)
    db = bd.DeviceBatch.from_host(b)
    ws = bd.Workspace()
    g = bd.DeviceGraph(b.n_atoms, 64, 16, 64)
    bd.build_graph(hp, db, g, ws)
    return hp, db, g, ws


def _check_step(bd, b, params, targets, d, T, name, delta=None, magmom=False):
    ohp = om.HParams(d=d, n_layers=T, conservative=True, magmom=magmom)
    graph = og.build_graph(b.atom_ptr, b.pos, b.lattice)
    rl, rg = autodiff.loss_and_grad(ohp, b, graph, params.astype(np.float64), targets, delta=delta)
    hp, db, g, ws = _setup(bd, b, d, T, magmom=magmom)
    loss, grad = bd.step(hp, db, g, _dev(params), [_dev(x) for x in targets], ws, huber_delta=delta or 0.0)
    lv = float(loss.cpu().numpy()[0])
    assert abs(lv - rl) <= 1e-5 + 1e-4 * abs(rl), (name, lv, rl)
    _assert_grad(grad.cpu().numpy(), rg, ohp, name)


def test_step_cubic8(bd):
    b, params, targets, d, T = synth.workload_inputs("cubic8")
    _check_step(bd, b, params, targets, d, T, "cubic8 conservative step")


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_step_random_batches(bd, seed):
    b = synth.random_crystals(seed=500 + seed, n_struct=1 + seed, n_lo=2, n_hi=12, rho=(0.06, 0.12))
    params = synth.make_params(64, 3, seed=(12, 1, seed))
    targets = synth.make_targets(b, seed=(12, 2, seed))
    _check_step(bd, b, params, targets, 64, 3, "random%d conservative step" % seed, delta=0.1 if seed == 1 else None)


def test_step_magmom_head(bd):
    b = synth.random_crystals(seed=21, n_struct=2, n_lo=3, n_hi=10)
    params = synth.make_params(64, 3, seed=(12, 1, 7), magmom=True)
    targets = synth.make_targets(b, seed=(12, 2, 7), magmom=True)
    _check_step(bd, b, params, targets, 64, 3, "magmom conservative step", magmom=True)
    _check_step(bd, b, params, targets, 64, 3, "magmom huber conservative step", delta=0.2, magmom=True)


def test_step_sparse_cells(bd):
    """Edges but no bonds (one atom in a 5 A cube: B = A = 0), bonds but no
    angles (a dimer: one bond per atom), and an isolated atom (E = 0)."""
    params = synth.make_params(64, 2, seed=(8, 1, 0))
    cells = [
        ("edges only", synth.make_custom_batch([np.eye(3) * 5.0], [np.zeros((1, 3))], [np.array([14])])),
        ("dimer", synth.make_custom_batch([np.eye(3) * 10.0], [np.array([[0.0, 0.0, 0.0], [0.15, 0.0, 0.0]])],
                                          [np.array([8, 8])])),
        ("no edges", synth.make_custom_batch([np.eye(3) * 13.0], [np.zeros((1, 3))], [np.array([26])])),
    ]
    for k, (name, b) in enumerate(cells):
        g = og.build_graph(b.atom_ptr, b.pos, b.lattice)
        print(name, "E B A =", len(g["edge_dst"]), len(g["bond_edge"]), len(g["angle_b2"]), flush=True)
        _check_step(bd, b, params, synth.make_targets(b, seed=(8, 2, k)), 64, 2, name + " conservative step")


def test_step_d128_single_layer(bd):
    b = synth.random_crystals(seed=11, n_struct=2, n_lo=4, n_hi=10)
    _check_step(bd, b, synth.make_params(128, 2, seed=(7, 1, 1)), synth.make_targets(b, seed=(7, 2, 1)), 128, 2,
                "d128 conservative step")
    _check_step(bd, b, synth.make_params(64, 1, seed=(7, 1, 3)), synth.make_targets(b, seed=(7, 2, 3)), 64, 1,
                "T1 conservative step")


def test_backward_random_output_gradients(bd):
    """chgnet_backward after chgnet_forward: the gradient of sum(dE E) +
    sum(dF F) + sum(dS sigma) for random dE, dF, dS."""
    import torch

    b, params, _, d, T = synth.workload_inputs("cubic8")
    rng = np.random.default_rng(5)
    dE = rng.standard_normal(b.n_struct)
    dF = rng.standard_normal((b.n_atoms, 3))
    dS = rng.standard_normal((b.n_struct, 3, 3))
    ohp = om.HParams(d=d, n_layers=T, conservative=True)
    graph = og.build_graph(b.atom_ptr, b.pos, b.lattice)
    p64 = torch.tensor(params.astype(np.float64), requires_grad=True)
    E, F, S, _, _ = autodiff.outputs(ohp, b, graph, p64, create_graph=True)
    tot = (E * torch.tensor(dE)).sum() + (F * torch.tensor(dF)).sum() + (S * torch.tensor(dS)).sum()
    (rg,) = torch.autograd.grad(tot, p64)
    hp, db, g, ws = _setup(bd, b, d, T)
    p = _dev(params)
    bd.forward(hp, db, g, p, ws)
    f32 = lambda x: _dev(x.astype(np.float32))
    grad = bd.backward(hp, db, g, p, f32(dE), f32(dF), f32(dS), ws)
    _assert_grad(grad.cpu().numpy(), rg.numpy(), ohp, "cubic8 conservative backward")


@pytest.mark.parametrize("workload,sample", [("triclinic40", [3, 22]), ("wide128", [5, 77])])
def test_full_size_sampled_structures(bd, workload, sample):
    import torch

    from gpu_helpers import subset_batch

    b, params, _, d, T = synth.workload_inputs(workload)
    rng = np.random.default_rng(9)
    dE = np.zeros(b.n_struct)
    dF = np.zeros((b.n_atoms, 3))
    dS = np.zeros((b.n_struct, 3, 3))
    sb = subset_batch(b, sample)
    sE = rng.standard_normal(len(sample))
    sF = rng.standard_normal((sb.n_atoms, 3))
    sS = rng.standard_normal((len(sample), 3, 3))
    o = 0
    for k, s in enumerate(sample):
        a0, a1 = b.atom_ptr[s], b.atom_ptr[s + 1]
        dE[s], dS[s] = sE[k], sS[k]
        dF[a0:a1] = sF[o:o + a1 - a0]
        o += a1 - a0
    ohp = om.HParams(d=d, n_layers=T, conservative=True)
    graph = og.build_graph(sb.atom_ptr, sb.pos, sb.lattice)
    p64 = torch.tensor(params.astype(np.float64), requires_grad=True)
    E, F, S, _, _ = autodiff.outputs(ohp, sb, graph, p64, create_graph=True)
    tot = (E * torch.tensor(sE)).sum() + (F * torch.tensor(sF)).sum() + (S * torch.tensor(sS)).sum()
    (rg,) = torch.autograd.grad(tot, p64)
    hp, db, g, ws = _setup(bd, b, d, T)
    p = _dev(params)
    bd.forward(hp, db, g, p, ws)
    f32 = lambda x: _dev(x.astype(np.float32))
    grad = bd.backward(hp, db, g, p, f32(dE), f32(dF), f32(dS), ws)
    _assert_grad(grad.cpu().numpy(), rg.numpy(), ohp, workload + " sampled conservative backward")


def _check_step_seq(bd, b, params, targets, d, T, name, delta=None, magmom=False):
    ohp = om.HParams(d=d, n_layers=T, conservative=True, magmom=magmom, sequential=True)
    graph = og.build_graph(b.atom_ptr, b.pos, b.lattice)
    rl, rg = autodiff.loss_and_grad(ohp, b, graph, params.astype(np.float64), targets, delta=delta)
    hp, db, g, ws = _setup(bd, b, d, T, magmom=magmom, sequential=True)
    loss, grad = bd.step(hp, db, g, _dev(params), [_dev(x) for x in targets], ws, huber_delta=delta or 0.0)
    lv = float(loss.cpu().numpy()[0])
    assert abs(lv - rl) <= 1e-5 + 1e-4 * abs(rl), (name, lv, rl)
    _assert_grad(grad.cpu().numpy(), rg, ohp, name)


def test_eq10_block_step(bd):
    """Training through the conservative readout with the reference block of
    Eq. (10) (bond conv on v^{t+1}, angle update on v^{t+1} and e^{t+1}):
    cubic8, random batches (one with Huber), the moment head and d = 128."""
    b, params, targets, d, T = synth.workload_inputs("cubic8")
    _check_step_seq(bd, b, params, targets, d, T, "cubic8 eq10 conservative step")
    for seed in (0, 1):
        br = synth.random_crystals(seed=520 + seed, n_struct=2 + seed, n_lo=2, n_hi=12, rho=(0.06, 0.12))
        _check_step_seq(bd, br, synth.make_params(64, 3, seed=(13, 1, seed)), synth.make_targets(br, seed=(13, 2, seed)),
                        64, 3, "random%d eq10 conservative step" % seed, delta=0.1 if seed else None)
    bm = synth.random_crystals(seed=23, n_struct=2, n_lo=3, n_hi=10)
    _check_step_seq(bd, bm, synth.make_params(64, 2, seed=(13, 1, 7), magmom=True),
                    synth.make_targets(bm, seed=(13, 2, 7), magmom=True), 64, 2, "magmom eq10 conservative step",
                    magmom=True)
    _check_step_seq(bd, bm, synth.make_params(128, 2, seed=(13, 1, 9)), synth.make_targets(bm, seed=(13, 2, 9)), 128, 2,
                    "d128 eq10 conservative step")


def test_eq10_block_backward_random_output_gradients(bd):
    """chgnet_backward with the Eq. (10) block and random output gradients
    against autograd's second derivatives of sum(dE E) + sum(dF F) + sum(dS sigma)."""
    import torch

    b = synth.random_crystals(seed=31, n_struct=2, n_lo=4, n_hi=12)
    d, T = 64, 3
    params = synth.make_params(d, T, seed=(14, 1, 0))
    ohp = om.HParams(d=d, n_layers=T, conservative=True, sequential=True)
    rng = np.random.default_rng(4)
    dE = rng.standard_normal(b.n_struct)
    dF = rng.standard_normal((b.n_atoms, 3))
    dS = rng.standard_normal((b.n_struct, 3, 3))
    graph = og.build_graph(b.atom_ptr, b.pos, b.lattice)
    p64 = torch.tensor(params.astype(np.float64), requires_grad=True)
    E, F, S, _, _ = autodiff.outputs(ohp, b, graph, p64, create_graph=True)
    tot = (E * torch.tensor(dE)).sum() + (F * torch.tensor(dF)).sum() + (S * torch.tensor(dS)).sum()
    (rg,) = torch.autograd.grad(tot, p64)
    hp, db, g, ws = _setup(bd, b, d, T, sequential=True)
    p = _dev(params)
    bd.forward(hp, db, g, p, ws)
    f32 = lambda x: _dev(x.astype(np.float32))
    grad = bd.backward(hp, db, g, p, f32(dE), f32(dF), f32(dS), ws)
    _assert_grad(grad.cpu().numpy(), rg.numpy(), ohp, "eq10 conservative backward")


def test_step_bitwise_reproducible(bd):
    """Training through the conservative readout twice on the same inputs:
    the loss and every gradient entry are bitwise equal (every sum of the
    dual-number path runs in a fixed order)."""
    b, params, targets, d, T = synth.workload_inputs("triclinic40")
    hp, db, g, ws = _setup(bd, b, d, T)
    p = _dev(params)
    tg = [_dev(x) for x in targets]
    l1, g1 = bd.step(hp, db, g, p, tg, ws)
    l1, g1 = l1.cpu().numpy().copy(), g1.cpu().numpy().copy()
    l2, g2 = bd.step(hp, db, g, p, tg, ws)
    assert np.array_equal(l1, l2.cpu().numpy())
    assert np.array_equal(g1, g2.cpu().numpy())
