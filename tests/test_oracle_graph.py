"""Pins of the oracle's graph construction (atom graph, bond graph, angles).

The counts of lattice translations inside a sphere are computed here by exact
integer arithmetic on the lattice's integer coordinates (an independent
method: no fp32 predicate, no image-range pruning), and the two hand-countable
simple-cubic cases are stored as golden values."""
import itertools
import json
import math
import os

import numpy as np
import pytest

from oracle import graph
from paper_2412_20796_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _one_atom(L):
    return np.array([0, 1], np.int32), np.zeros((1, 3), np.float32), np.asarray(L, np.float32)[None]


def _count_integer_points(scale2, rc, parity=None):
    """#{k in Z^3 \\ 0 : scale2 * |k|^2 < rc^2}, optionally with a parity rule."""
    lim = int(math.ceil(rc / math.sqrt(scale2))) + 1
    n = 0
    for k in itertools.product(range(-lim, lim + 1), repeat=3):
        if k == (0, 0, 0):
            continue
        if parity == "even_sum" and sum(k) % 2:
            continue
        if parity == "same_parity" and len({x % 2 for x in k}) != 1:
            continue
        if scale2 * (k[0] ** 2 + k[1] ** 2 + k[2] ** 2) < rc * rc:
            n += 1
    return n


def test_golden_simple_cubic():
    with open(os.path.join(GOLDEN, "simple_cubic_counts.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        g = graph.build_graph(*_one_atom(np.eye(3) * c["a"]))
        assert len(g["edge_dst"]) == c["edges"], c
        assert len(g["bond_edge"]) == c["bonds"], c
        assert len(g["angle_b2"]) == c["angles"], c
        if c["angles"]:
            img = g["edge_img"][g["bond_edge"]].astype(float) * c["a"]
            b1 = np.repeat(np.arange(len(g["bond_edge"])), np.diff(g["angle_ptr"]))
            cosang = (img[b1] * img[g["angle_b2"]]).sum(1) / (c["a"] ** 2)
            assert int(np.isclose(cosang, 0.0).sum()) == c["angles_90"]
            assert int(np.isclose(cosang, -1.0).sum()) == c["angles_180"]


@pytest.mark.parametrize(
    "kind,a",
    [("sc", 1.7), ("sc", 2.5), ("sc", 3.3), ("fcc", 4.0), ("fcc", 3.1), ("bcc", 3.0), ("bcc", 2.7)],
)
def test_lattice_point_counts(kind, a):
    """One-atom primitive cells: every edge is a lattice translation, so
    counts equal the number of lattice points within the cutoffs."""
    if kind == "sc":
        L, scale2, par = np.eye(3) * a, a * a, None
    elif kind == "fcc":  # primitive vectors (a/2)(0,1,1) etc.; points (a/2)k, sum(k) even
        L, scale2, par = (a / 2) * (np.ones((3, 3)) - np.eye(3)), (a / 2) ** 2, "even_sum"
    else:  # bcc primitive vectors (a/2)(-1,1,1) etc.; points (a/2)k, k all same parity
        L, scale2, par = (a / 2) * (np.ones((3, 3)) - 2 * np.eye(3)), (a / 2) ** 2, "same_parity"
    g = graph.build_graph(*_one_atom(L))
    ne = _count_integer_points(scale2, 6.0, par)
    nb = _count_integer_points(scale2, 3.0, par)
    assert len(g["edge_dst"]) == ne
    assert len(g["bond_edge"]) == nb
    assert len(g["angle_b2"]) == nb * (nb - 1)
    # every edge is a self-image; its reverse is the negated translation
    e = np.arange(len(g["edge_dst"]))
    assert (g["edge_dst"] == 0).all()
    np.testing.assert_array_equal(g["edge_img"][g["edge_rev"]], -g["edge_img"])
    assert (g["edge_rev"][g["edge_rev"]] == e).all()


def _scalar_bruteforce(atom_ptr, pos, lat, rc, reach=6):
    """Pure-Python enumeration over a very wide image box, scalar fp32."""
    out = []
    f32 = np.float32
    for s in range(len(atom_ptr) - 1):
        L = lat[s]
        for i in range(atom_ptr[s], atom_ptr[s + 1]):
            for j in range(atom_ptr[s], atom_ptr[s + 1]):
                for n in itertools.product(range(-reach, reach + 1), repeat=3):
                    if i == j and n == (0, 0, 0):
                        continue
                    dl = []
                    for c in range(3):
                        sc = f32(f32(f32(n[0]) * L[0, c]) + f32(f32(n[1]) * L[1, c])) + f32(f32(n[2]) * L[2, c])
                        dl.append(f32(f32(pos[j, c] + f32(sc)) - pos[i, c]))
                    d2 = f32(f32(dl[0] * dl[0]) + f32(dl[1] * dl[1])) + f32(dl[2] * dl[2])
                    if d2 < f32(rc * rc):
                        out.append((i, j) + tuple(n))
    return out


def test_scalar_bruteforce_small_triclinic():
    b = synth.random_crystals(seed=3, n_struct=2, n_lo=2, n_hi=3, rho=(0.09, 0.12))
    g = graph.build_graph(b.atom_ptr, b.pos, b.lattice)
    src = np.repeat(np.arange(b.n_atoms), np.diff(g["edge_ptr"]))
    got = [(int(src[e]), int(g["edge_dst"][e])) + tuple(int(x) for x in g["edge_img"][e]) for e in range(len(src))]
    want = _scalar_bruteforce(b.atom_ptr, b.pos, b.lattice, 6.0)
    assert got == sorted(want)  # canonical order = (i, j, n1, n2, n3) lexicographic
    assert max(abs(x) for t in got for x in t[2:]) < 6  # the box was wide enough


def test_structure_and_index_invariants():
    b = synth.random_crystals(seed=1, n_struct=3, n_lo=4, n_hi=12)
    g = graph.build_graph(b.atom_ptr, b.pos, b.lattice)
    N = b.n_atoms
    src = np.repeat(np.arange(N), np.diff(g["edge_ptr"]))
    struct = np.repeat(np.arange(b.n_struct), np.diff(b.atom_ptr))
    assert (struct[src] == struct[g["edge_dst"]]).all()
    rev = g["edge_rev"]
    assert (rev[rev] == np.arange(len(rev))).all()
    assert (g["edge_dst"][rev] == src).all()
    np.testing.assert_array_equal(g["edge_img"][rev], -g["edge_img"])
    # bonds: subsequence of edges, shorter than 3 A, grouped per source atom
    be = g["bond_edge"]
    assert (np.diff(be) > 0).all()
    assert (g["edge_d2"][be] < 9.0).all()
    assert (np.delete(g["edge_d2"], be) >= 9.0).all()
    k = np.diff(g["bond_ptr"])
    assert (src[be] == np.repeat(np.arange(N), k)).all()
    assert g["angle_ptr"][-1] == (k * (k - 1)).sum() == len(g["angle_b2"])
    b1 = np.repeat(np.arange(len(be)), np.diff(g["angle_ptr"]))
    assert (b1 != g["angle_b2"]).all()
    assert (src[be[b1]] == src[be[g["angle_b2"]]]).all()
    # bond graph is symmetric under reversal
    assert (g["edge_d2"][rev[be]] < 9.0).all()


def test_supercell_replication():
    b = synth.random_crystals(seed=5, n_struct=1, n_lo=6, n_hi=6)
    L = b.lattice[0].astype(np.float64)
    frac = b.pos.astype(np.float64) @ np.linalg.inv(L)
    L2 = L.copy()
    L2[0] *= 2
    frac2 = np.concatenate([frac * [0.5, 1, 1], (frac + [1, 0, 0]) * [0.5, 1, 1]])
    b2 = synth.make_custom_batch([L2], [frac2], [np.concatenate([b.Z, b.Z])])
    b1 = synth.make_custom_batch([L], [frac], [b.Z])
    g1 = graph.build_graph(b1.atom_ptr, b1.pos, b1.lattice)
    g2 = graph.build_graph(b2.atom_ptr, b2.pos, b2.lattice)
    n = b1.n_atoms
    c1 = np.diff(g1["edge_ptr"])
    c2 = np.diff(g2["edge_ptr"])
    np.testing.assert_array_equal(c2[:n], c1)
    np.testing.assert_array_equal(c2[n:], c1)
    assert len(g2["angle_b2"]) == 2 * len(g1["angle_b2"])
    for i in range(n):
        d1 = np.sort(g1["edge_d2"][g1["edge_ptr"][i]:g1["edge_ptr"][i + 1]])
        d2 = np.sort(g2["edge_d2"][g2["edge_ptr"][i]:g2["edge_ptr"][i + 1]])
        np.testing.assert_allclose(d1, d2, rtol=1e-5)


def test_sampled_rows_match_full_build():
    b = synth.random_crystals(seed=2, n_struct=2, n_lo=5, n_hi=9)
    g = graph.build_graph(b.atom_ptr, b.pos, b.lattice)
    rows = graph.build_graph(b.atom_ptr, b.pos, b.lattice, atoms=[0, 3, b.n_atoms - 1])
    for i, (dst, img) in rows.items():
        lo, hi = g["edge_ptr"][i], g["edge_ptr"][i + 1]
        np.testing.assert_array_equal(dst, g["edge_dst"][lo:hi])
        np.testing.assert_array_equal(img, g["edge_img"][lo:hi])
