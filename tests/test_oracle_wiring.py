"""Pins of the interaction-block wiring (Eq. 4-6 with the Eq. 11 inputs).

Three atoms in a large cubic box (no periodic image within 6 A): atom 1 is
bonded to atoms 0 and 2 (2.5 A and 2.8 A, 120 degrees apart), atoms 0 and 2
are 4.6 A apart (an edge, not a bond). The width is d = 2 and each GatedMLP
reads a single block of its concatenated input through the weights
core = +x, gate = -x (bias 0, LayerNorm scale 1 and shift 0). A LayerNorm
over two values x = (x1, x2) gives (s, -s) with s = h / sqrt(h^2 + eps),
h = (x1 - x2) / 2, so the gate of a block value x is, by hand,

    phi(x) = (SiLU(s) sigmoid(-s), SiLU(-s) sigmoid(s)),

and phi(0) = 0. Atom 1's element row is (1, -1); atoms 0 and 2 have zero
rows. Which block is read, and over which edges or angles a message is
summed, then decides which sums are zero and what the others equal:

* atom conv, Eq. (4): m_i = sum over the edges (i, j) leaving i of
  e^a_ij * phi([v_i, v_j, e_ij]);
* bond conv, Eq. (5): mu_b = sum over the angles (b, b') whose first bond is
  b, at the centre atom i, of e^b_b * e^b_b' * phi([v_i, e_b, e_b', a]);
* angle update, Eq. (6): a' = a + phi([v_i, e_b, e_b', a]).

A block swap (v_i for v_j, e_b for e_b'), a sum over entering instead of
leaving edges, or the destination atom in place of the centre each make one
of these checks fail."""
import math

import numpy as np
import pytest

from oracle import graph as og
from oracle import model as om
from paper_2412_20796_amd import synth

D = 2
EPS = 1e-5


def _phi_hand(x):
    x1, x2 = float(x[0]), float(x[1])
    h = (x1 - x2) / 2.0
    s = h / math.sqrt(h * h + EPS)
    sig = lambda t: 1.0 / (1.0 + math.exp(-t))
    return np.array([s * sig(s) * sig(-s), -s * sig(-s) * sig(s)])


def _batch():
    c = 2.8 * math.cos(math.radians(60.0)), 2.8 * math.sin(math.radians(60.0))
    pos = np.array([[5.0, 5.0, 5.0], [7.5, 5.0, 5.0], [7.5 + c[0], 5.0 + c[1], 5.0]], np.float32)
    return synth.Batch(np.array([0, 3], np.int32), pos, (np.eye(3, dtype=np.float32) * 20.0)[None],
                       np.array([1, 2, 3], np.int32))


def _params(hp, block, module):
    """Zero weights except the embeddings and one block of one GatedMLP."""
    rng = np.random.default_rng(5)
    lay, n = om.layout(hp)
    p = np.zeros(n)

    def put(name, val):
        off, shape = lay[name]
        p[off:off + int(np.prod(shape))] = np.asarray(val, float).reshape(-1)

    put("W_Z", np.zeros((94, D)))
    off, _ = lay["W_Z"]
    p[off + 1 * D:off + 2 * D] = [1.0, -1.0]  # element Z = 2 (atom 1)
    put("f_a", np.pi * np.arange(1, hp.n_rbf + 1))
    put("f_b", np.pi * np.arange(1, hp.n_rbf + 1))
    put("W_e", rng.uniform(-1, 1, (hp.n_rbf, 2 * D)))
    put("b_e0", rng.uniform(-1, 1, D))
    put("W_eb", rng.uniform(-1, 1, (hp.n_rbf, D)))
    put("W_th", rng.uniform(-1, 1, (hp.n_fourier, D)))
    put("b_th", rng.uniform(-1, 1, D))
    for t in range(hp.n_layers):
        for m in ("av_", "be_", "an_"):
            pre = "L%d_%s" % (t, m)
            if pre + "g_c" not in lay:
                continue
            put(pre + "g_c", np.ones(D))
            put(pre + "g_g", np.ones(D))
        put("L%d_av_Wo" % t, np.eye(D))
        put("L%d_be_Wo" % t, np.eye(D))
    rows = 3 * D if module == "av_" else 4 * D
    W = np.zeros((rows, 2 * D))
    W[block * D:(block + 1) * D, :D] = np.eye(D)
    W[block * D:(block + 1) * D, D:] = -np.eye(D)
    put("L0_%sW" % module, W)
    return p


def _run(block, module, T=1):
    hp = om.HParams(d=D, n_layers=T)
    b = _batch()
    g = og.build_graph(b.atom_ptr, b.pos, b.lattice)
    _, _, _, cache = om.forward(hp, b, g, _params(hp, block, module))
    src = np.repeat(np.arange(3), np.diff(g["edge_ptr"]))
    edge = {(int(src[e]), int(g["edge_dst"][e])): e for e in range(len(src))}
    bond = {(int(src[e]), int(g["edge_dst"][e])): k for k, e in enumerate(g["bond_edge"])}
    return cache, edge, bond


def test_geometry_of_the_fixture():
    _, edge, bond = _run(0, "av_")
    assert sorted(edge) == [(0, 1), (0, 2), (1, 0), (1, 2), (2, 0), (2, 1)]
    assert sorted(bond) == [(0, 1), (1, 0), (1, 2), (2, 1)]


def test_atom_conv_reads_the_destination_block_over_leaving_edges():
    cache, edge, _ = _run(1, "av_")  # rows of v_j
    m, ea = cache["layers"][0]["m"], cache["ea"]
    p1 = _phi_hand([1.0, -1.0])
    np.testing.assert_allclose(m[0], ea[edge[0, 1]] * p1, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(m[2], ea[edge[2, 1]] * p1, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(m[1], 0.0, atol=1e-15)


def test_atom_conv_reads_the_source_block():
    cache, edge, _ = _run(0, "av_")  # rows of v_i
    m, ea = cache["layers"][0]["m"], cache["ea"]
    p1 = _phi_hand([1.0, -1.0])
    np.testing.assert_allclose(m[1], (ea[edge[1, 0]] + ea[edge[1, 2]]) * p1, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(m[[0, 2]], 0.0, atol=1e-15)


def test_atom_conv_edge_block_and_update():
    cache, edge, _ = _run(2, "av_")  # rows of e_ij
    L0 = cache["layers"][0]
    m, ea, e = L0["m"], cache["ea"], L0["e"]
    for i in range(3):
        want = sum(ea[edge[i, j]] * _phi_hand(e[edge[i, j]]) for j in range(3) if (i, j) in edge)
        np.testing.assert_allclose(m[i], want, rtol=1e-12, atol=1e-15)
    # v' = v + m Wo + bo with Wo = I, bo = 0 (T = 1: v^T)
    np.testing.assert_allclose(cache["vT"], L0["v"] + m, rtol=1e-12, atol=1e-15)


def test_bond_conv_reads_the_centre_atom():
    cache, _, bond = _run(0, "be_")  # rows of v_i, the centre
    mu, eb = cache["layers"][0]["mu"], cache["eb"]
    p1 = _phi_hand([1.0, -1.0])
    np.testing.assert_allclose(mu[bond[1, 0]], eb[bond[1, 0]] * eb[bond[1, 2]] * p1, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(mu[bond[1, 2]], eb[bond[1, 2]] * eb[bond[1, 0]] * p1, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(mu[[bond[0, 1], bond[2, 1]]], 0.0, atol=1e-15)


@pytest.mark.parametrize("block,which", [(1, "first"), (2, "second")])
def test_bond_conv_bond_blocks(block, which):
    cache, edge, bond = _run(block, "be_")  # rows of e_b (first bond) or e_b' (second)
    L0 = cache["layers"][0]
    mu, eb, e = L0["mu"], cache["eb"], L0["e"]
    for b, other in (((1, 0), (1, 2)), ((1, 2), (1, 0))):
        read = b if which == "first" else other
        want = eb[bond[b]] * eb[bond[other]] * _phi_hand(e[edge[read]])
        np.testing.assert_allclose(mu[bond[b]], want, rtol=1e-12, atol=1e-15)
    # e' = e + mu Wo + bo on the bonds, the other edges unchanged
    e1 = cache["eT"]
    for (i, j), k in bond.items():
        np.testing.assert_allclose(e1[edge[i, j]], e[edge[i, j]] + mu[k], rtol=1e-12, atol=1e-15)
    for pair in ((0, 2), (2, 0)):
        np.testing.assert_array_equal(e1[edge[pair]], e[edge[pair]])


def test_angle_update_reads_the_angle_block():
    cache, _, _ = _run(3, "an_", T=2)  # rows of a, layer 0 (T = 2 keeps its angle update)
    a0, a1 = cache["layers"][0]["a"], cache["layers"][1]["a"]
    assert a0.shape == (2, D)
    for k in range(2):
        np.testing.assert_allclose(a1[k], a0[k] + _phi_hand(a0[k]), rtol=1e-12, atol=1e-15)
