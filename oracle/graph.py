"""Oracle: periodic atom graph G^a, bond graph G^b and the angle list.

Definitions (Sec. II-B (1) of the paper; cutoffs from Sec. IV, "Dataset"):

* G^a holds every directed edge (i, j, n): atoms i and j of the same crystal,
  n an integer lattice translation, (i, j, n) != (i, i, 0), whose separation
  r_j + n L - r_i is shorter than the atom-graph cutoff (6 A).
* G^b is the subset of G^a edges shorter than the bond-graph cutoff (3 A).
* An angle is an ordered pair (b, b') of distinct G^b edges leaving the same
  centre atom.

Reading (the paper does not say how the cutoff test is rounded): the test is
an fp32 expression evaluated in one fixed orientation of each pair. The two
directions (i, j, n) and (j, i, -n) of a pair describe one separation; the
canonical one is (i, j, n) with i < j, or, for i = j, with n
lexicographically positive (first non-zero component > 0). With (p, q, m)
the canonical orientation of the edge being tested,

    s_c  = ((m1*L1c) + (m2*L2c)) + (m3*L3c)
    dl_c = (r_qc + s_c) - r_pc
    D2   = ((dl_x*dl_x) + (dl_y*dl_y)) + (dl_z*dl_z)

with one IEEE round-to-nearest per operation and no fused multiply-add, and
an edge exists iff D2 < rc*rc (strict). Both directions therefore get the
same D2, so an edge's reverse always exists (the plain expression
(r_j + s) - r_i rounds differently from (r_i - s) - r_j, and near the
cutoff one direction can pass while the other fails). This makes the edge
set exactly reproducible. Every translation satisfying the test is kept (no
truncation of the image range); the per-pair enumeration range below is
generous.

Canonical order: edges grouped by source atom i (CSR), then by j, then by
(n1, n2, n3) lexicographically. rev(i, j, n) = (j, i, -n). Bonds keep G^a
order. Angles at a centre with bonds b_1 < ... < b_k are the k(k-1) ordered
pairs (b, b'), b != b', ordered by (b, b').
"""
from __future__ import annotations

import numpy as np


def interplanar_spacings(L):
    """Distance between adjacent lattice planes along each axis (fp64)."""
    L = np.asarray(L, dtype=np.float64)
    vol = abs(np.linalg.det(L))
    return vol / np.linalg.norm(np.cross(L[[1, 2, 0]], L[[2, 0, 1]]), axis=1)


def fp32_d2(ri, rj, n, L):
    """The fp32 expression ((r_j + s) - r_i)^2 summed over x, y, z, with
    s = n L, vectorised over leading axes of rj and n (one orientation).

    ri: float32 [..., 3] or [3]; rj: float32 [..., 3]; n: int [..., 3];
    L: float32 [3, 3]. Every operation is a separate float32 ufunc, so each
    rounds once."""
    nf = n.astype(np.float32)
    L = L.astype(np.float32)
    ri = np.asarray(ri, np.float32)
    dl = []
    for c in range(3):
        s = (nf[..., 0] * L[0, c] + nf[..., 1] * L[1, c]) + nf[..., 2] * L[2, c]
        dl.append((rj[..., c] + s) - ri[..., c])
    d2 = (dl[0] * dl[0] + dl[1] * dl[1]) + dl[2] * dl[2]
    assert d2.dtype == np.float32
    return d2


def is_canonical(i, j, n):
    """True where (i, j, n) is the canonical orientation of its pair: i < j,
    or i = j and n lexicographically positive. Vectorised over i, j, n[..., 3]."""
    n = np.asarray(n)
    lexpos = (n[..., 0] > 0) | ((n[..., 0] == 0) & ((n[..., 1] > 0) | ((n[..., 1] == 0) & (n[..., 2] > 0))))
    i = np.asarray(i)
    j = np.asarray(j)
    return (i < j) | ((i == j) & lexpos)


def pair_d2(i, j, n, pos32, L):
    """The cutoff test's D2 of edges (i, j, n): the fp32 expression evaluated
    in the canonical orientation of each pair, so that D2(i, j, n) equals
    D2(j, i, -n) bit for bit. i, j int [...]; n int [..., 3]."""
    i = np.asarray(i)
    j = np.asarray(j)
    n = np.asarray(n)
    canon = is_canonical(i, j, n)
    p = np.where(canon, i, j)
    q = np.where(canon, j, i)
    m = np.where(canon[..., None], n, -n)
    return fp32_d2(pos32[p], pos32[q], m, L)


def _edges_of_atom(i, a0, a1, pos32, L32, frac, h, rc):
    """All (j, n, D2) with D2 < rc^2 for source atom i, in canonical order.

    A translation n can only pass if |df_a + n_a| <= (rc + slack) / h_a on
    every axis (the component of a displacement along the normal of a lattice
    plane bounds its length), so each pair (i, j) is tested on every integer
    n_a in that interval, with 0.5 A of slack for the fp32 rounding."""
    rc2 = np.float32(rc * rc)
    js = np.arange(a0, a1)
    df = frac[a0:a1] - frac[i]  # [n_s, 3], fp64
    reach = (rc + 0.5) / h
    lo = np.ceil(-df - reach).astype(np.int64)  # [n_s, 3]
    cnt = np.floor(-df + reach).astype(np.int64) - lo + 1
    kmax = cnt.max(axis=0)
    grid = np.stack(np.meshgrid(*[np.arange(k) for k in kmax], indexing="ij"), axis=-1).reshape(-1, 3)
    Nimg = lo[:, None, :] + grid[None, :, :]  # [n_s, G, 3]
    valid = (grid[None, :, :] < cnt[:, None, :]).all(axis=2)
    J = np.broadcast_to(js[:, None], valid.shape)[valid]
    Nimg = Nimg[valid]
    d2 = pair_d2(np.full(J.shape, i), J, Nimg, pos32, L32)
    keep = d2 < rc2
    keep &= ~((J == i) & (Nimg == 0).all(axis=1))
    J, Nimg, d2 = J[keep], Nimg[keep], d2[keep]
    order = np.lexsort((Nimg[:, 2], Nimg[:, 1], Nimg[:, 0], J))
    return J[order], Nimg[order], d2[order]


def build_graph(atom_ptr, pos, lattice, r_atom=6.0, r_bond=3.0, atoms=None):
    """Build the graph of a batch.

    atom_ptr int [S+1]; pos float32 [N,3] Cartesian; lattice float32 [S,3,3]
    (rows are lattice vectors). If ``atoms`` is given, only those source
    atoms' edge rows are built (returned as a dict atom -> (dst, img)); this
    is how full-size graphs are sampled.

    Returns a dict of int32 arrays: edge_ptr [N+1], edge_dst [E],
    edge_img [E,3], edge_rev [E], bond_ptr [N+1], bond_edge [B],
    angle_ptr [B+1], angle_b2 [A]; and float32 edge_d2 [E]."""
    atom_ptr = np.asarray(atom_ptr, dtype=np.int64)
    pos32 = np.asarray(pos, dtype=np.float32)
    lat32 = np.asarray(lattice, dtype=np.float32)
    S = lat32.shape[0]
    N = pos32.shape[0]
    frac = np.empty((N, 3))
    hs = []
    for s in range(S):
        L = lat32[s].astype(np.float64)
        a0, a1 = atom_ptr[s], atom_ptr[s + 1]
        frac[a0:a1] = pos32[a0:a1].astype(np.float64) @ np.linalg.inv(L)
        hs.append(interplanar_spacings(L))
    struct_of = np.repeat(np.arange(S), np.diff(atom_ptr))

    if atoms is not None:
        rows = {}
        for i in atoms:
            s = struct_of[i]
            J, Nimg, _ = _edges_of_atom(i, atom_ptr[s], atom_ptr[s + 1], pos32, lat32[s], frac, hs[s], r_atom)
            rows[int(i)] = (J.astype(np.int32), Nimg.astype(np.int32))
        return rows

    dst, img, d2s, counts = [], [], [], np.zeros(N, dtype=np.int64)
    for i in range(N):
        s = struct_of[i]
        J, Nimg, d2 = _edges_of_atom(i, atom_ptr[s], atom_ptr[s + 1], pos32, lat32[s], frac, hs[s], r_atom)
        dst.append(J)
        img.append(Nimg)
        d2s.append(d2)
        counts[i] = J.shape[0]
    edge_ptr = np.zeros(N + 1, dtype=np.int64)
    edge_ptr[1:] = np.cumsum(counts)
    edge_dst = np.concatenate(dst) if N else np.zeros(0, np.int64)
    edge_img = np.concatenate(img) if N else np.zeros((0, 3), np.int64)
    edge_d2 = np.concatenate(d2s) if N else np.zeros(0, np.float32)
    E = edge_dst.shape[0]
    src = np.repeat(np.arange(N), counts)

    # reverse map through a dictionary on (src, dst, image)
    index = {(int(src[e]), int(edge_dst[e]), *map(int, edge_img[e])): e for e in range(E)}
    edge_rev = np.array(
        [index[(int(edge_dst[e]), int(src[e]), *map(int, -edge_img[e]))] for e in range(E)], dtype=np.int64
    )

    is_bond = edge_d2 < np.float32(r_bond * r_bond)
    bond_edge = np.nonzero(is_bond)[0]
    k = np.array([is_bond[edge_ptr[i]:edge_ptr[i + 1]].sum() for i in range(N)], dtype=np.int64)
    bond_ptr = np.zeros(N + 1, dtype=np.int64)
    bond_ptr[1:] = np.cumsum(k)
    B = bond_edge.shape[0]
    angle_ptr = np.zeros(B + 1, dtype=np.int64)
    b2 = []
    for i in range(N):
        for p in range(bond_ptr[i], bond_ptr[i + 1]):
            others = [q for q in range(bond_ptr[i], bond_ptr[i + 1]) if q != p]
            angle_ptr[p + 1] = angle_ptr[p] + len(others)
            b2.extend(others)
    return {
        "edge_ptr": edge_ptr.astype(np.int32),
        "edge_dst": edge_dst.astype(np.int32),
        "edge_img": edge_img.astype(np.int32).reshape(-1, 3),
        "edge_rev": edge_rev.astype(np.int32),
        "bond_ptr": bond_ptr.astype(np.int32),
        "bond_edge": bond_edge.astype(np.int32),
        "angle_ptr": angle_ptr.astype(np.int32),
        "angle_b2": np.asarray(b2, dtype=np.int32),
        "edge_d2": edge_d2.astype(np.float32),
    }
