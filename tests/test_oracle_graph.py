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
    """Pure-Python enumeration over a very wide image box, scalar fp32, each
    pair's separation taken in its canonical orientation (lower atom index
    first; for an atom's own images, the translation whose first non-zero
    component is positive)."""
    out = []
    f32 = np.float32
    for s in range(len(atom_ptr) - 1):
        L = lat[s]
        for i in range(atom_ptr[s], atom_ptr[s + 1]):
            for j in range(atom_ptr[s], atom_ptr[s + 1]):
                for n in itertools.product(range(-reach, reach + 1), repeat=3):
                    if i == j and n == (0, 0, 0):
                        continue
                    first = next(x for x in n if x != 0) if any(n) else 0
                    if i < j or (i == j and first > 0):
                        p, q, m = i, j, n
                    else:
                        p, q, m = j, i, tuple(-x for x in n)
                    dl = []
                    for c in range(3):
                        sc = f32(f32(f32(m[0]) * L[0, c]) + f32(f32(m[1]) * L[1, c])) + f32(f32(m[2]) * L[2, c])
                        dl.append(f32(f32(pos[q, c] + f32(sc)) - pos[p, c]))
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


def _edge_tuples(g):
    src = np.repeat(np.arange(len(g["edge_ptr"]) - 1), np.diff(g["edge_ptr"]))
    return [(int(src[e]), int(g["edge_dst"][e])) + tuple(int(x) for x in g["edge_img"][e]) for e in range(len(src))]


def _assert_reverse_total(g):
    """Every edge (i, j, n) has its reverse (j, i, -n), and edge_rev names it."""
    src = np.repeat(np.arange(len(g["edge_ptr"]) - 1), np.diff(g["edge_ptr"]))
    rev = g["edge_rev"]
    assert (rev[rev] == np.arange(len(rev))).all()
    assert (g["edge_dst"][rev] == src).all() and (src[rev] == g["edge_dst"]).all()
    np.testing.assert_array_equal(g["edge_img"][rev], -g["edge_img"])
    ed = set(_edge_tuples(g))
    assert all((t[1], t[0], -t[2], -t[3], -t[4]) in ed for t in ed)
    # bond graph closed under reversal, D2 equal in both directions
    be = set(g["bond_edge"].tolist())
    assert all(int(rev[b]) in be for b in be)
    np.testing.assert_array_equal(g["edge_d2"][rev], g["edge_d2"])


def test_golden_reverse_pair_cell():
    """A pair 1 fp32 ulp inside the cutoff in one orientation and exactly on it
    in the other (golden fixture): both directions are edges."""
    from fractions import Fraction

    with open(os.path.join(GOLDEN, "reverse_pair_cell.json")) as f:
        c = json.load(f)
    a = np.float32(c["lattice_a"])
    pos = np.asarray(c["pos"], np.float32)
    g = graph.build_graph(np.array([0, 2]), pos, (np.eye(3, dtype=np.float32) * a)[None])
    _assert_reverse_total(g)
    got = set(_edge_tuples(g))
    for t in c["boundary_edges"]:
        assert tuple(t) in got, t
    assert len(got) == c["edges"]
    # away from the boundary, membership follows exact rational arithmetic
    A = Fraction(float(a))
    P = [[Fraction(float(x)) for x in r] for r in pos]
    away = 0
    for i in range(2):
        for j in range(2):
            for n in itertools.product(range(-3, 4), repeat=3):
                if i == j and n == (0, 0, 0):
                    continue
                d2 = sum((P[j][k] + n[k] * A - P[i][k]) ** 2 for k in range(3))
                if abs(d2 - 36) > Fraction(1, 1000):
                    assert ((i, j) + n in got) == (d2 < 36), (i, j, n)
                    away += d2 < 36
    assert away == c["edges_away_from_boundary"]


@pytest.mark.parametrize("kind", ["atom", "bond", "self"])
def test_boundary_sweeps_keep_reverse_edges(kind):
    """Pairs stepped ulp by ulp across the 6 A and 3 A cutoffs (through a
    lattice translation, and an atom's own images): every edge has its
    reverse, the bonds are closed under reversal, and the edge set equals a
    scalar brute force. The sweep includes pairs whose two one-orientation
    evaluations fall on opposite sides of the cutoff, so a test in one
    orientation only would fail here."""
    b = synth.boundary_batch(kind)
    g = graph.build_graph(b.atom_ptr, b.pos, b.lattice)
    _assert_reverse_total(g)
    assert _edge_tuples(g) == sorted(_scalar_bruteforce(b.atom_ptr, b.pos, b.lattice, 6.0, reach=2))
    rc2 = np.float32(9.0 if kind == "bond" else 36.0)
    split = 0
    for s in range(b.n_struct):
        a0, a1 = b.atom_ptr[s], b.atom_ptr[s + 1]
        for i in range(a0, a1):
            for j in range(a0, a1):
                n = np.array([[1, 0, 0]])
                fwd = graph.fp32_d2(b.pos[i], b.pos[j][None], n, b.lattice[s])[0]
                bwd = graph.fp32_d2(b.pos[j], b.pos[i][None], -n, b.lattice[s])[0]
                split += (fwd < rc2) != (bwd < rc2)
    assert split > 0


@pytest.mark.parametrize("seed", range(4))
def test_random_cells_reverse_total(seed):
    """No guard band: random triclinic cells, every edge has its reverse."""
    b = synth.random_crystals(seed=300 + seed, n_struct=4, n_lo=2, n_hi=24, rho=(0.06, 0.12))
    _assert_reverse_total(graph.build_graph(b.atom_ptr, b.pos, b.lattice))
