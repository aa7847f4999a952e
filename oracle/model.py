"""Oracle: FastCHGNet forward, loss, hand-written backward and Adam (fp64).

Everything here follows the paper's definitions literally:

* Feature embedding, Eq. (2): element table, smooth radial Bessel basis
  (sRBF) of the edge length, Fourier basis of the bond angle, linear maps.
* Interaction block, Eq. (3)-(6) with the dependency-free inputs of Eq. (11):
  the atom conv, bond conv and angle update of layer t all read layer-t
  features.
* GatedMLP (Sec. II-B (3)): phi(x) = SiLU(LN(Fc_c(x))) * sigmoid(LN(Fc_g(x))),
  applied to the literal concatenated input.
* Energy output (Sec. II-B (4)); Force head, Eq. (7); Stress head, Eq. (9).
* Loss with the paper's prefactors (Sec. IV, "Parameters Setting").

Readings where the paper is silent or garbled (fixed here and in the GPU
library alike):

* Envelope: Eq. (12) and Eq. (13) as printed do not vanish at the cutoff; the
  DimeNet polynomial envelope (which the paper cites for sRBF) is used:
  u(x) = 1 - (p+1)(p+2)/2 x^p + p(p+2) x^(p+1) - p(p+1)/2 x^(p+2), p = 8.
* sRBF_c(r)_n = sqrt(2/c) sin(f_n r / c) / r * u(r/c), with trainable
  frequencies f_n initialised to n*pi; one basis at the 6 A cutoff feeds
  e^0 and e^a, another at 3 A feeds e^b (bond graph).
* FT(theta) = [1/sqrt(2 pi), cos(m theta)/sqrt(pi) (m=1..M), sin(m theta)/sqrt(pi)
  (m=1..M)], 2M+1 = 31; theta = atan2(|r_ij x r_ik|, r_ij . r_ik).
* e^a and e^b linear maps have no bias; e^0 and a^0 have one.
* Bond features are directed; bond conv updates G^b edges only.
* The last layer's angle update is omitted (its output feeds nothing).
* Head MLPs are d -> d -> d -> out with SiLU; the force head output is a
  scalar per edge, symmetrised over the reverse edge, times the unit vector
  from i to the image of j.
* Stress head: sigma_s = (1/V_s) sum_i sum_ab c_i,ab u_a u_b^T, u_a the unit
  lattice vectors, c_i the 9 outputs of the stress MLP.
* Loss: prefactor-weighted mean squared errors of per-atom energy, force
  components and stress components; optionally the Huber loss of Sec. IV
  (h(r) = r^2/2 for |r| <= delta, delta (|r| - delta/2) beyond), whose delta
  the paper does not state (a caller's choice).
* Magnetic-moment head (Sec. II-B; Sec. IV lists magmom among the
  predictions but gives no formula): m_i = |v^T_i w_m + b_m|, a linear map of
  the final atom features whose absolute value is the moment's magnitude;
  d|x|/dx at 0 is taken as 0. Its loss term averages over the N atoms.
* Interaction-block order: the default is Eq. (11) (all three modules read
  layer-t features). HParams.sequential selects the reference block of
  Eq. (10): the bond conv reads v^{t+1}, the angle update reads v^{t+1} and
  the updated bond features e^{t+1} (Eq. (5), (6)).
* Conservative readout (HParams.conservative; the reference CHGNet output
  layer, Sec. II-B (4)): F_i = -dE/dr_i and sigma = (1/V) dE/d(eps) for the
  homogeneous strain r -> (I + eps) r of positions and lattice, replacing the
  force and stress heads (whose weights are then unused). E depends on the
  positions only through the edge vectors r_e = r_j + n L - r_i (lengths in
  the radial bases, bond-pair angles in the Fourier basis), so with
  g_e = dE/dr_e: F_i = sum over edges leaving i of g_e minus the sum over
  edges entering i, and sigma = (1/V) sum_e g_e r_e^T. d(theta)/dr is
  undefined for collinear bond pairs (|r1 x r2| = 0); it is taken as 0 there.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

N_ELEMENTS = 94
LN_EPS = 1e-5


@dataclass(frozen=True)
class HParams:
    d: int = 64
    n_layers: int = 4
    n_rbf: int = 31
    n_fourier: int = 31
    envelope_p: int = 8
    r_atom: float = 6.0
    r_bond: float = 3.0
    magmom: bool = False        # magnetic-moment head
    sequential: bool = False    # Eq. (10) block instead of Eq. (11)
    conservative: bool = False  # F and sigma as derivatives of E


# ---------------------------------------------------------------------------
# Flat parameter layout (the order documented with the C interface).
# ---------------------------------------------------------------------------

def layout(hp: HParams):
    d, T, R, K = hp.d, hp.n_layers, hp.n_rbf, hp.n_fourier
    ent = [("W_Z", (N_ELEMENTS, d)), ("f_a", (R,)), ("f_b", (R,)), ("W_e", (R, 2 * d)),
           ("b_e0", (d,)), ("W_eb", (R, d)), ("W_th", (K, d)), ("b_th", (d,))]

    def gm(prefix, fan_in_rows):
        return [(prefix + "W", (fan_in_rows, 2 * d)), (prefix + "b", (2 * d,)),
                (prefix + "g_c", (d,)), (prefix + "b_c", (d,)), (prefix + "g_g", (d,)), (prefix + "b_g", (d,))]

    for t in range(T):
        ent += gm("L%d_av_" % t, 3 * d) + [("L%d_av_Wo" % t, (d, d)), ("L%d_av_bo" % t, (d,))]
        ent += gm("L%d_be_" % t, 4 * d) + [("L%d_be_Wo" % t, (d, d)), ("L%d_be_bo" % t, (d,))]
        if t < T - 1:
            ent += gm("L%d_an_" % t, 4 * d)
    for h, o in (("E", 1), ("F", 1), ("S", 9)):
        ent += [(h + "_W1", (d, d)), (h + "_b1", (d,)), (h + "_W2", (d, d)), (h + "_b2", (d,)),
                (h + "_W3", (d, o)), (h + "_b3", (o,))]
    if hp.magmom:
        ent += [("M_W", (d, 1)), ("M_b", (1,))]
    out, off = {}, 0
    for name, shape in ent:
        n = int(np.prod(shape))
        out[name] = (off, shape)
        off += n
    return out, off


def param_count(hp: HParams) -> int:
    return layout(hp)[1]


def unpack(hp: HParams, flat):
    lay, total = layout(hp)
    flat = np.asarray(flat)
    assert flat.shape == (total,), (flat.shape, total)
    return {k: flat[o:o + int(np.prod(s))].reshape(s) for k, (o, s) in lay.items()}


# ---------------------------------------------------------------------------
# Elementary functions (textbook definitions).
# ---------------------------------------------------------------------------

def sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


def silu(x):
    return x * sigmoid(x)


def dsilu(x):
    s = sigmoid(x)
    return s * (1.0 + x * (1.0 - s))


def envelope(x, p):
    """DimeNet polynomial envelope u(x); u(0)=1, u(1)=u'(1)=u''(1)=0."""
    return (1.0 - (p + 1) * (p + 2) / 2.0 * x ** p + p * (p + 2) * x ** (p + 1)
            - p * (p + 1) / 2.0 * x ** (p + 2))


def srbf(r, freq, cutoff, p):
    """Smooth radial Bessel basis, [n_edges, n_rbf]."""
    r = np.asarray(r, dtype=np.float64)[:, None]
    return math.sqrt(2.0 / cutoff) * np.sin(freq[None, :] * r / cutoff) / r * envelope(r / cutoff, p)


def srbf_dfreq(r, freq, cutoff, p):
    """d sRBF_n / d f_n (elementwise), [n_edges, n_rbf]."""
    r = np.asarray(r, dtype=np.float64)[:, None]
    return math.sqrt(2.0 / cutoff) * np.cos(freq[None, :] * r / cutoff) / cutoff * envelope(r / cutoff, p)


def envelope_dx(x, p):
    """u'(x) from differentiating each term of the polynomial."""
    return (-(p + 1) * (p + 2) / 2.0 * p * x ** (p - 1) + p * (p + 2) * (p + 1) * x ** p
            - p * (p + 1) / 2.0 * (p + 2) * x ** (p + 1))


def srbf_dr(r, freq, cutoff, p):
    """d sRBF_n / d r (product rule on sin(f r / c) * (1/r) * u(r/c)), [n_edges, n_rbf]."""
    r = np.asarray(r, dtype=np.float64)[:, None]
    a = freq[None, :] * r / cutoff
    x = r / cutoff
    return math.sqrt(2.0 / cutoff) * (np.cos(a) * freq[None, :] / cutoff / r * envelope(x, p)
                                      - np.sin(a) / (r * r) * envelope(x, p)
                                      + np.sin(a) / r * envelope_dx(x, p) / cutoff)


def fourier_dtheta(theta, n_fourier):
    """d FT / d theta, [n_angles, n_fourier]."""
    m = (n_fourier - 1) // 2
    ks = np.arange(1, m + 1)[None, :]
    th = np.asarray(theta, dtype=np.float64)[:, None]
    return np.concatenate([np.zeros((th.shape[0], 1)), -ks * np.sin(ks * th) / math.sqrt(math.pi),
                           ks * np.cos(ks * th) / math.sqrt(math.pi)], axis=1)


def fourier(theta, n_fourier):
    m = (n_fourier - 1) // 2
    ks = np.arange(1, m + 1)[None, :]
    th = np.asarray(theta, dtype=np.float64)[:, None]
    return np.concatenate([np.full((th.shape[0], 1), 1.0 / math.sqrt(2 * math.pi)),
                           np.cos(ks * th) / math.sqrt(math.pi), np.sin(ks * th) / math.sqrt(math.pi)], axis=1)


def layernorm(z, g, b):
    mu = z.mean(axis=1, keepdims=True)
    var = ((z - mu) ** 2).mean(axis=1, keepdims=True)
    xhat = (z - mu) / np.sqrt(var + LN_EPS)
    return g * xhat + b, xhat, 1.0 / np.sqrt(var + LN_EPS)


def gated_mlp(x, P, prefix, d):
    """phi(x) and the saved pre-activation z = x W + b."""
    z = x @ P[prefix + "W"] + P[prefix + "b"]
    yc, _, _ = layernorm(z[:, :d], P[prefix + "g_c"], P[prefix + "b_c"])
    yg, _, _ = layernorm(z[:, d:], P[prefix + "g_g"], P[prefix + "b_g"])
    return silu(yc) * sigmoid(yg), z


def gated_mlp_backward(dphi, x, z, P, prefix, d, G):
    """Accumulate parameter grads into G; return dL/dx."""
    zc, zg = z[:, :d], z[:, d:]
    yc, xc, rc = layernorm(zc, P[prefix + "g_c"], P[prefix + "b_c"])
    yg, xg, rg = layernorm(zg, P[prefix + "g_g"], P[prefix + "b_g"])
    sc, sg = silu(yc), sigmoid(yg)
    dyc = dphi * sg * dsilu(yc)
    dyg = dphi * sc * sg * (1.0 - sg)

    def ln_back(dy, xhat, rstd, gname, bname):
        G[gname] += (dy * xhat).sum(axis=0)
        G[bname] += dy.sum(axis=0)
        dx = dy * P[gname]
        return rstd * (dx - dx.mean(axis=1, keepdims=True) - xhat * (dx * xhat).mean(axis=1, keepdims=True))

    dz = np.concatenate([ln_back(dyc, xc, rc, prefix + "g_c", prefix + "b_c"),
                         ln_back(dyg, xg, rg, prefix + "g_g", prefix + "b_g")], axis=1)
    G[prefix + "W"] += x.T @ dz
    G[prefix + "b"] += dz.sum(axis=0)
    return dz @ P[prefix + "W"].T


def mlp3(x, P, h):
    h1 = x @ P[h + "_W1"] + P[h + "_b1"]
    a1 = silu(h1)
    h2 = a1 @ P[h + "_W2"] + P[h + "_b2"]
    a2 = silu(h2)
    return a2 @ P[h + "_W3"] + P[h + "_b3"], (h1, a1, h2, a2)


def mlp3_backward(do, x, cache, P, h, G):
    h1, a1, h2, a2 = cache
    G[h + "_W3"] += a2.T @ do
    G[h + "_b3"] += do.sum(axis=0)
    dh2 = (do @ P[h + "_W3"].T) * dsilu(h2)
    G[h + "_W2"] += a1.T @ dh2
    G[h + "_b2"] += dh2.sum(axis=0)
    dh1 = (dh2 @ P[h + "_W2"].T) * dsilu(h1)
    G[h + "_W1"] += x.T @ dh1
    G[h + "_b1"] += dh1.sum(axis=0)
    return dh1 @ P[h + "_W1"].T


def seg_sum(values, index, n):
    out = np.zeros((n,) + values.shape[1:], dtype=np.float64)
    np.add.at(out, index, values)
    return out


# ---------------------------------------------------------------------------
# Geometry and indices derived from the graph.
# ---------------------------------------------------------------------------

def derived(batch, graph):
    atom_ptr = np.asarray(batch.atom_ptr, dtype=np.int64)
    N = int(atom_ptr[-1])
    S = atom_ptr.shape[0] - 1
    edge_ptr = graph["edge_ptr"].astype(np.int64)
    src = np.repeat(np.arange(N), np.diff(edge_ptr))
    dst = graph["edge_dst"].astype(np.int64)
    img = graph["edge_img"].astype(np.float64)
    struct = np.repeat(np.arange(S), np.diff(atom_ptr))
    pos = np.asarray(batch.pos, dtype=np.float64)
    L = np.asarray(batch.lattice, dtype=np.float64)
    rvec = pos[dst] + np.einsum("ea,eac->ec", img, L[struct[src]]) - pos[src]
    dist = np.linalg.norm(rvec, axis=1)
    bond_edge = graph["bond_edge"].astype(np.int64)
    bond_ptr = graph["bond_ptr"].astype(np.int64)
    angle_ptr = graph["angle_ptr"].astype(np.int64)
    B = bond_edge.shape[0]
    b1 = np.repeat(np.arange(B), np.diff(angle_ptr))
    b2 = graph["angle_b2"].astype(np.int64)
    centre = src[bond_edge[b1]] if B else np.zeros(0, np.int64)
    ra, rb = rvec[bond_edge[b1]], rvec[bond_edge[b2]]
    theta = np.arctan2(np.linalg.norm(np.cross(ra, rb), axis=1), (ra * rb).sum(axis=1))
    return dict(N=N, S=S, E=dst.shape[0], B=B, A=b1.shape[0], src=src, dst=dst, struct=struct,
                rvec=rvec, dist=dist, bond_edge=bond_edge, bond_ptr=bond_ptr, b1=b1, b2=b2,
                centre=centre, theta=theta, rev=graph["edge_rev"].astype(np.int64),
                n_per=np.diff(atom_ptr).astype(np.float64), L=L)


# ---------------------------------------------------------------------------
# Forward.
# ---------------------------------------------------------------------------

def forward(hp: HParams, batch, graph, params):
    """Returns (energy [S], forces [N,3], stress [S,3,3], cache); with the
    magnetic-moment head, cache["magmom"] holds the moments [N]."""
    P = unpack(hp, np.asarray(params, dtype=np.float64))
    g = derived(batch, graph)
    d, T = hp.d, hp.n_layers
    N, S = g["N"], g["S"]
    src, dst, be, b1, b2, ctr = g["src"], g["dst"], g["bond_edge"], g["b1"], g["b2"], g["centre"]

    # Eq. (2): embeddings
    Z = np.asarray(batch.Z, dtype=np.int64)
    v = P["W_Z"][Z - 1]
    rbf_a = srbf(g["dist"], P["f_a"], hp.r_atom, hp.envelope_p)
    e0ea = rbf_a @ P["W_e"]
    e = e0ea[:, :d] + P["b_e0"]
    ea = e0ea[:, d:]
    rbf_b = srbf(g["dist"][be], P["f_b"], hp.r_bond, hp.envelope_p)
    eb = rbf_b @ P["W_eb"]
    ft = fourier(g["theta"], hp.n_fourier)
    a = ft @ P["W_th"] + P["b_th"]

    layers = []
    for t in range(T):
        pre = "L%d_" % t
        # Eq. (4): atom conv
        fv = np.concatenate([v[src], v[dst], e], axis=1)
        phiv, zv = gated_mlp(fv, P, pre + "av_", d)
        m = seg_sum(ea * phiv, src, N)
        v_new = v + m @ P[pre + "av_Wo"] + P[pre + "av_bo"]
        # Eq. (5): bond conv on [v_i, e_ij, e_ik, a_ijk], v = v^t under
        # Eq. (11), v^{t+1} under Eq. (10)
        vb = v_new if hp.sequential else v
        fa = np.concatenate([vb[ctr], e[be[b1]], e[be[b2]], a], axis=1)
        phie, ze = gated_mlp(fa, P, pre + "be_", d)
        ssum = seg_sum(eb[b2] * phie, b1, g["B"])
        mu = eb * ssum
        e_new = e.copy()
        e_new[be] += mu @ P[pre + "be_Wo"] + P[pre + "be_bo"]
        # Eq. (6): angle update; Eq. (11) reuses the bond-conv input, Eq. (10)
        # reads v^{t+1} and e^{t+1}
        za, a_new, fan = None, a, fa
        if t < T - 1:
            if hp.sequential:
                fan = np.concatenate([v_new[ctr], e_new[be[b1]], e_new[be[b2]], a], axis=1)
            phia, za = gated_mlp(fan, P, pre + "an_", d)
            a_new = a + phia
        layers.append(dict(v=v, e=e, a=a, fv=fv, zv=zv, phiv=phiv, m=m, fa=fa, ze=ze, phie=phie,
                           ssum=ssum, mu=mu, za=za, fan=fan))
        v, e, a = v_new, e_new, a_new

    # Energy output (Sec. II-B (4)): sum over atoms of an MLP of v^T
    oE, cE = mlp3(v, P, "E")
    energy = seg_sum(oE, g["struct"], S)[:, 0]
    # Force head, Eq. (7): scalar per edge, symmetrised, times unit vector
    mF, cF = mlp3(e, P, "F")
    nE = 0.5 * (mF[:, 0] + mF[g["rev"], 0])
    xhat = g["rvec"] / g["dist"][:, None]
    forces = seg_sum(nE[:, None] * xhat, src, N)
    # Stress head, Eq. (9)
    cS, cSc = mlp3(v, P, "S")
    Csum = seg_sum(cS, g["struct"], S).reshape(S, 3, 3)
    U = g["L"] / np.linalg.norm(g["L"], axis=2, keepdims=True)
    vol = np.abs(np.linalg.det(g["L"]))
    stress = np.einsum("sab,sax,sby->sxy", Csum, U, U) / vol[:, None, None]

    # Magnetic moments: |v^T w_m + b_m| per atom
    oM = magmom = None
    if hp.magmom:
        oM = (v @ P["M_W"] + P["M_b"])[:, 0]
        magmom = np.abs(oM)

    cache = dict(P=P, g=g, Zidx=Z - 1, rbf_a=rbf_a, rbf_b=rbf_b, ft=ft, ea=ea, eb=eb, layers=layers, vT=v, eT=e,
                 cE=cE, cF=cF, cSc=cSc, xhat=xhat, U=U, vol=vol, oM=oM, magmom=magmom)
    if hp.conservative:
        forces, stress = conservative_readout(hp, cache)
    return energy, forces, stress, cache


def conservative_readout(hp, cache):
    """F = -dE/dr and sigma = (1/V) dE/d(eps) through the backward of E."""
    P, g = cache["P"], cache["g"]
    N, S = g["N"], g["S"]
    _, gi = backward(hp, cache, np.ones(S), np.zeros((N, 3)), np.zeros((S, 3, 3)), inputs=True)
    be, b1, b2, rvec, dist = g["bond_edge"], g["b1"], g["b2"], g["rvec"], g["dist"]
    xhat = rvec / dist[:, None]
    # radial bases: dE/d|r_e| along r_e / |r_e|
    gd = (gi["drbf_a"] * srbf_dr(dist, P["f_a"], hp.r_atom, hp.envelope_p)).sum(axis=1)
    gvec = gd[:, None] * xhat
    gdb = (gi["drbf_b"] * srbf_dr(dist[be], P["f_b"], hp.r_bond, hp.envelope_p)).sum(axis=1)
    np.add.at(gvec, be, gdb[:, None] * xhat[be])
    # angular basis: theta = atan2(|r1 x r2|, r1 . r2);
    # d theta / d r1 = (c r1 / |r1|^2 - r2) / s, and symmetrically for r2
    gth = (gi["dft"] * fourier_dtheta(g["theta"], hp.n_fourier)).sum(axis=1)
    r1, r2 = rvec[be[b1]], rvec[be[b2]]
    c = (r1 * r2).sum(axis=1)
    sn = np.linalg.norm(np.cross(r1, r2), axis=1)
    ok = sn > 0
    inv = np.where(ok, 1.0 / np.where(ok, sn, 1.0), 0.0)[:, None]
    d1 = (c[:, None] * r1 / (r1 * r1).sum(axis=1, keepdims=True) - r2) * inv
    d2 = (c[:, None] * r2 / (r2 * r2).sum(axis=1, keepdims=True) - r1) * inv
    np.add.at(gvec, be[b1], gth[:, None] * d1)
    np.add.at(gvec, be[b2], gth[:, None] * d2)
    # r_e = r_dst + n L - r_src
    forces = seg_sum(gvec, g["src"], N) - seg_sum(gvec, g["dst"], N)
    sig = seg_sum(np.einsum("ea,eb->eab", gvec, rvec), g["struct"][g["src"]], S)
    return forces, sig / cache["vol"][:, None, None]


# ---------------------------------------------------------------------------
# Loss.
# ---------------------------------------------------------------------------

def huber(r, delta):
    """Huber's loss of residuals r: r^2/2 inside [-delta, delta], linear with
    slope delta outside; and its derivative clip(r, -delta, delta)."""
    r = np.asarray(r, dtype=np.float64)
    inside = np.abs(r) <= delta
    return (np.where(inside, 0.5 * r * r, delta * (np.abs(r) - 0.5 * delta)),
            np.where(inside, r, delta * np.sign(r)))


def _pointwise(r, delta):
    """(loss, derivative) per residual: squared error, or Huber if delta."""
    r = np.asarray(r, dtype=np.float64)
    if delta is None:
        return r * r, 2.0 * r
    return huber(r, delta)


def loss_and_grads(energy, forces, stress, n_per, E_t, F_t, S_t, w=(2.0, 1.5, 0.1), delta=None):
    """Weighted mean of per-atom energy, force-component and stress-component
    errors (squared, or Huber with threshold delta) and its gradient."""
    S = energy.shape[0]
    N = forces.shape[0]
    le, ge = _pointwise(energy / n_per - E_t, delta)
    lf, gf = _pointwise(forces - F_t, delta)
    ls, gs = _pointwise(stress - S_t, delta)
    loss = w[0] * np.mean(le) + w[1] * np.mean(lf) + w[2] * np.mean(ls)
    dE = w[0] * ge / n_per / S
    dF = w[1] * gf / (3 * N)
    dS = w[2] * gs / (9 * S)
    return loss, dE, dF, dS


def magmom_loss(magmom, M_t, w=0.1, delta=None):
    """Weighted mean over atoms of the magnetic-moment error and its gradient."""
    lm, gm = _pointwise(np.asarray(magmom, dtype=np.float64) - M_t, delta)
    return w * np.mean(lm), w * gm / magmom.shape[0]


# ---------------------------------------------------------------------------
# Backward (first order, weights only).
# ---------------------------------------------------------------------------

def backward(hp: HParams, cache, dE, dF, dS, dM=None, inputs=False):
    """Gradient of <dE,E> + <dF,F> + <dS,sigma> (+ <dM,magmom>) w.r.t. every
    parameter (flat), with the direct force and stress heads. With inputs,
    also the gradients with respect to the two radial bases and the angular
    basis: (flat, dict(drbf_a, drbf_b, dft))."""
    P, g = cache["P"], cache["g"]
    d, T = hp.d, hp.n_layers
    N, S, B = g["N"], g["S"], g["B"]
    src, dst, be, b1, b2, ctr = g["src"], g["dst"], g["bond_edge"], g["b1"], g["b2"], g["centre"]
    G = {k: np.zeros_like(v) for k, v in P.items()}
    dE = np.asarray(dE, dtype=np.float64)
    dF = np.asarray(dF, dtype=np.float64)
    dS = np.asarray(dS, dtype=np.float64)

    # heads
    dv = mlp3_backward(dE[g["struct"]][:, None], cache["vT"], cache["cE"], P, "E", G)
    dC = np.einsum("sxy,sax,sby->sab", dS, cache["U"], cache["U"]) / cache["vol"][:, None, None]
    dv += mlp3_backward(dC.reshape(S, 9)[g["struct"]], cache["vT"], cache["cSc"], P, "S", G)
    if hp.magmom and dM is not None:
        gm = np.asarray(dM, dtype=np.float64) * np.sign(cache["oM"])
        G["M_W"] += cache["vT"].T @ gm[:, None]
        G["M_b"] += gm.sum()
        dv += gm[:, None] * P["M_W"][:, 0][None, :]
    dn = (dF[src] * cache["xhat"]).sum(axis=1)
    dm = 0.5 * (dn + dn[g["rev"]])
    de = mlp3_backward(dm[:, None], cache["eT"], cache["cF"], P, "F", G)

    dea = np.zeros_like(cache["ea"])
    deb = np.zeros_like(cache["eb"])
    da = None
    ea, eb = cache["ea"], cache["eb"]
    seq = hp.sequential
    for t in reversed(range(T)):
        pre = "L%d_" % t
        Ls = cache["layers"][t]
        # dv, de, da: gradients with respect to v^{t+1}, e^{t+1}, a^{t+1}
        da_in = np.zeros_like(Ls["a"]) if da is None else da.copy()
        if seq and t < T - 1:
            # Eq. (10): the angle update read v^{t+1} and e^{t+1}
            dfan = gated_mlp_backward(da, Ls["fan"], Ls["za"], P, pre + "an_", d, G)
            dv = dv + seg_sum(dfan[:, :d], ctr, N)
            de = de + seg_sum(dfan[:, d:2 * d], be[b1], g["E"]) + seg_sum(dfan[:, 2 * d:3 * d], be[b2], g["E"])
            da_in += dfan[:, 3 * d:]
        de_in = de.copy()
        # e'_b = e_b + mu Wo + bo (bonds only)
        deb_rows = de[be]
        dmu = deb_rows @ P[pre + "be_Wo"].T
        G[pre + "be_Wo"] += Ls["mu"].T @ deb_rows
        G[pre + "be_bo"] += deb_rows.sum(axis=0)
        # mu_b = eb_b * sum_{alpha: b1=b} eb_b2 * phi_e
        deb += dmu * Ls["ssum"]
        dphie = dmu[b1] * eb[b1] * eb[b2]
        deb += seg_sum(dmu[b1] * eb[b1] * Ls["phie"], b2, B)
        dfa = gated_mlp_backward(dphie, Ls["fa"], Ls["ze"], P, pre + "be_", d, G)
        if not seq and t < T - 1:
            dfa = dfa + gated_mlp_backward(da, Ls["fa"], Ls["za"], P, pre + "an_", d, G)
        dv_ctr = seg_sum(dfa[:, :d], ctr, N)
        if seq:
            dv = dv + dv_ctr  # the bond conv read v^{t+1}
        de_in += seg_sum(dfa[:, d:2 * d], be[b1], g["E"])
        de_in += seg_sum(dfa[:, 2 * d:3 * d], be[b2], g["E"])
        da_in += dfa[:, 3 * d:]
        # v' = v + m Wo + bo
        dv_in = dv.copy() if seq else dv + dv_ctr
        dmsg = dv @ P[pre + "av_Wo"].T
        G[pre + "av_Wo"] += Ls["m"].T @ dv
        G[pre + "av_bo"] += dv.sum(axis=0)
        # m_i = sum_e ea_e * phi_v
        dphiv = dmsg[src] * ea
        dea += dmsg[src] * Ls["phiv"]
        dfv = gated_mlp_backward(dphiv, Ls["fv"], Ls["zv"], P, pre + "av_", d, G)
        dv_in += seg_sum(dfv[:, :d], src, N)
        dv_in += seg_sum(dfv[:, d:2 * d], dst, N)
        de_in += dfv[:, 2 * d:]
        dv, de, da = dv_in, de_in, da_in

    # embeddings
    G["W_Z"] += seg_sum(dv, cache["Zidx"], N_ELEMENTS)
    de0ea = np.concatenate([de, dea], axis=1)
    G["W_e"] += cache["rbf_a"].T @ de0ea
    G["b_e0"] += de.sum(axis=0)
    drbf_a = de0ea @ P["W_e"].T
    G["f_a"] += (drbf_a * srbf_dfreq(g["dist"], P["f_a"], hp.r_atom, hp.envelope_p)).sum(axis=0)
    G["W_eb"] += cache["rbf_b"].T @ deb
    drbf_b = deb @ P["W_eb"].T
    G["f_b"] += (drbf_b * srbf_dfreq(g["dist"][be], P["f_b"], hp.r_bond, hp.envelope_p)).sum(axis=0)
    G["W_th"] += cache["ft"].T @ da
    G["b_th"] += da.sum(axis=0)

    lay, total = layout(hp)
    flat = np.zeros(total)
    for k, (o, s) in lay.items():
        flat[o:o + int(np.prod(s))] = G[k].reshape(-1)
    if inputs:
        return flat, dict(drbf_a=drbf_a, drbf_b=drbf_b, dft=da @ P["W_th"].T)
    return flat


def adam(params, grad, m, v, lr, b1, b2, eps, t):
    """Kingma and Ba's Adam update (bias-corrected), step number t >= 1."""
    m = b1 * m + (1 - b1) * grad
    v = b2 * v + (1 - b2) * grad * grad
    mhat = m / (1 - b1 ** t)
    vhat = v / (1 - b2 ** t)
    return params - lr * mhat / (np.sqrt(vhat) + eps), m, v


def step(hp: HParams, batch, params, targets, w=(2.0, 1.5, 0.1), graph=None, delta=None, w_m=0.1):
    """Graph build, forward, loss, backward: (loss, grad, outputs). targets are
    (E, F, S) per-atom energy, forces, stress, plus magnetic moments M [N]
    when the head is on; delta selects the Huber loss; w_m weighs the moments."""
    from . import graph as graph_mod

    if hp.conservative:
        raise NotImplementedError("training through the conservative readout needs second derivatives")
    if graph is None:
        graph = graph_mod.build_graph(batch.atom_ptr, batch.pos, batch.lattice, hp.r_atom, hp.r_bond)
    energy, forces, stress, cache = forward(hp, batch, graph, params)
    loss, dE, dF, dS = loss_and_grads(energy, forces, stress, cache["g"]["n_per"], *targets[:3], w=w, delta=delta)
    dM = None
    outputs = (energy, forces, stress)
    if hp.magmom:
        lm, dM = magmom_loss(cache["magmom"], targets[3], w_m, delta)
        loss += lm
        outputs = outputs + (cache["magmom"],)
    grad = backward(hp, cache, dE, dF, dS, dM)
    return loss, grad, outputs, graph
