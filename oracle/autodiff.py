"""Oracle (test infrastructure; nothing in the GPU library imports it): an
independent PyTorch-CPU fp64 transcription of the model forward, with
derivatives taken by automatic differentiation instead of by hand.

It serves two purposes:

* a witness for the hand-written backward of oracle.model (the weight
  gradient of the loss with the direct force and stress heads) and for its
  conservative readout (F = -dE/dr, sigma = (1/V) dE/d(eps));
* the training gradient through the conservative readout (the reference
  CHGNet output layer of Sec. II-B (4)), which needs second derivatives:
  the loss depends on F = -dE/dr, so its weight gradient differentiates a
  derivative. autograd builds the graph of dE/dr (create_graph) and
  differentiates the loss through it.

The forward is written from the definitions (Eq. (2), (4)-(6) with the
inputs of Eq. (11) or Eq. (10), the GatedMLP of Sec. II-B (3), the heads of
Sec. II-B (4), Eq. (7)-(9)) and the same readings as oracle.model (see its
docstring); only the flat parameter layout (data, not arithmetic) is shared.
Strain convention: positions and lattice deform as r -> (I + eps) r, so an
edge vector r_e becomes (I + eps_s) r_e; sigma = (1/V) dE/d(eps). The angle
is theta = atan2(|r1 x r2|, r1 . r2); for collinear bond pairs (|r1 x r2| =
0) its derivative is undefined and taken as 0, as in oracle.model.
"""
from __future__ import annotations

import math

import numpy as np
import torch

from .model import layout

_LN_EPS = 1e-5
_DT = torch.float64


def _t(x, dtype=_DT):
    return torch.as_tensor(np.ascontiguousarray(x), dtype=dtype)


def _params(hp, flat):
    lay, total = layout(hp)
    assert flat.shape == (total,)
    return {k: flat[o:o + int(np.prod(s))].reshape(s) for k, (o, s) in lay.items()}


def _indices(batch, graph):
    """Integer structure of the graph: edge source/destination/structure,
    bonds, angles (first bond, second bond, centre)."""
    ap = np.asarray(batch.atom_ptr, dtype=np.int64)
    N, S = int(ap[-1]), ap.shape[0] - 1
    ep = graph["edge_ptr"].astype(np.int64)
    src = np.repeat(np.arange(N), np.diff(ep))
    bond_edge = graph["bond_edge"].astype(np.int64)
    angle_ptr = graph["angle_ptr"].astype(np.int64)
    B = bond_edge.shape[0]
    b1 = np.repeat(np.arange(B), np.diff(angle_ptr))
    b2 = graph["angle_b2"].astype(np.int64)
    struct = np.repeat(np.arange(S), np.diff(ap))
    return dict(N=N, S=S, src=src, dst=graph["edge_dst"].astype(np.int64), img=graph["edge_img"].astype(np.float64),
                rev=graph["edge_rev"].astype(np.int64), struct=struct, estruct=struct[src], bond_edge=bond_edge,
                b1=b1, b2=b2, n_per=np.diff(ap).astype(np.float64))


def _segsum(x, idx, n):
    out = torch.zeros((n,) + tuple(x.shape[1:]), dtype=x.dtype)
    return out.index_add(0, idx, x)


def _envelope(x, p):
    return 1.0 - (p + 1) * (p + 2) / 2.0 * x ** p + p * (p + 2) * x ** (p + 1) - p * (p + 1) / 2.0 * x ** (p + 2)


def _srbf(r, f, c, p):
    r = r[:, None]
    return math.sqrt(2.0 / c) * torch.sin(f[None, :] * r / c) / r * _envelope(r / c, p)


def _fourier(theta, K):
    M = (K - 1) // 2
    m = torch.arange(1, M + 1, dtype=_DT)[None, :]
    th = theta[:, None]
    return torch.cat([torch.full_like(th, 1.0 / math.sqrt(2.0 * math.pi)), torch.cos(m * th) / math.sqrt(math.pi),
                      torch.sin(m * th) / math.sqrt(math.pi)], dim=1)


def _ln(z, g, b):
    mu = z.mean(dim=1, keepdim=True)
    var = ((z - mu) ** 2).mean(dim=1, keepdim=True)
    return g * (z - mu) / torch.sqrt(var + _LN_EPS) + b


def _gated(x, P, pre, d):
    z = x @ P[pre + "W"] + P[pre + "b"]
    return torch.nn.functional.silu(_ln(z[:, :d], P[pre + "g_c"], P[pre + "b_c"])) * torch.sigmoid(
        _ln(z[:, d:], P[pre + "g_g"], P[pre + "b_g"]))


def _mlp(x, P, h):
    a1 = torch.nn.functional.silu(x @ P[h + "_W1"] + P[h + "_b1"])
    a2 = torch.nn.functional.silu(a1 @ P[h + "_W2"] + P[h + "_b2"])
    return a2 @ P[h + "_W3"] + P[h + "_b3"]


def forward(hp, batch, graph, params, pos=None, strain=None, ix=None):
    """(E [S], direct F [N,3], direct sigma [S,3,3], magmom [N] or None) as
    torch tensors; params, pos [N,3] and strain [S,3,3] may require grad."""
    ix = ix or _indices(batch, graph)
    P = _params(hp, params)
    d, T = hp.d, hp.n_layers
    N, S = ix["N"], ix["S"]
    src, dst, struct = (torch.as_tensor(ix[k]) for k in ("src", "dst", "struct"))
    be, b1, b2 = (torch.as_tensor(ix[k]) for k in ("bond_edge", "b1", "b2"))
    lat = _t(batch.lattice)
    pos = _t(batch.pos) if pos is None else pos
    # edge vectors r_e = (I + eps_s)(r_dst + n L - r_src)
    r = pos[dst] + torch.einsum("ea,eac->ec", _t(ix["img"]), lat[torch.as_tensor(ix["estruct"])]) - pos[src]
    if strain is not None:
        r = r + torch.einsum("eab,eb->ea", strain[torch.as_tensor(ix["estruct"])], r)
    dist = torch.sqrt((r * r).sum(dim=1))
    ctr = src[be[b1]]
    r1, r2 = r[be[b1]], r[be[b2]]
    cr = torch.linalg.cross(r1, r2)
    # |r1 x r2| with a zero derivative where it vanishes (collinear pairs,
    # such as a bond and its opposite self-image): d theta / d r = 0 there
    c2 = (cr * cr).sum(dim=1)
    pos_c2 = c2 > 0
    sn = torch.where(pos_c2, torch.sqrt(torch.where(pos_c2, c2, torch.ones_like(c2))), torch.zeros_like(c2))
    theta = torch.atan2(sn, (r1 * r2).sum(dim=1))

    # Eq. (2)
    v = P["W_Z"][torch.as_tensor(np.asarray(batch.Z, dtype=np.int64) - 1)]
    rbf = _srbf(dist, P["f_a"], hp.r_atom, hp.envelope_p)
    e = rbf @ P["W_e"][:, :d] + P["b_e0"]
    ea = rbf @ P["W_e"][:, d:]
    eb = _srbf(dist[be], P["f_b"], hp.r_bond, hp.envelope_p) @ P["W_eb"]
    a = _fourier(theta, hp.n_fourier) @ P["W_th"] + P["b_th"]
    B = be.shape[0]
    for t in range(T):
        pre = "L%d_" % t
        # Eq. (4)
        m = _segsum(ea * _gated(torch.cat([v[src], v[dst], e], dim=1), P, pre + "av_", d), src, N)
        v1 = v + m @ P[pre + "av_Wo"] + P[pre + "av_bo"]
        # Eq. (5)
        vb = v1 if hp.sequential else v
        phie = _gated(torch.cat([vb[ctr], e[be[b1]], e[be[b2]], a], dim=1), P, pre + "be_", d)
        mu = eb * _segsum(eb[b2] * phie, b1, B)
        e1 = e.index_add(0, be, mu @ P[pre + "be_Wo"] + P[pre + "be_bo"])
        # Eq. (6)
        a1 = a
        if t < T - 1:
            if hp.sequential:
                x = torch.cat([v1[ctr], e1[be[b1]], e1[be[b2]], a], dim=1)
            else:
                x = torch.cat([v[ctr], e[be[b1]], e[be[b2]], a], dim=1)
            a1 = a + _gated(x, P, pre + "an_", d)
        v, e, a = v1, e1, a1

    E = _segsum(_mlp(v, P, "E"), struct, S)[:, 0]
    mF = _mlp(e, P, "F")[:, 0]
    n = 0.5 * (mF + mF[torch.as_tensor(ix["rev"])])
    F = _segsum(n[:, None] * r / dist[:, None], src, N)
    U = lat / torch.linalg.norm(lat, dim=2, keepdim=True)
    vol = torch.abs(torch.linalg.det(lat))
    C = _segsum(_mlp(v, P, "S"), struct, S).reshape(S, 3, 3)
    sig = torch.einsum("sab,sax,sby->sxy", C, U, U) / vol[:, None, None]
    M = torch.abs((v @ P["M_W"] + P["M_b"])[:, 0]) if hp.magmom else None
    return E, F, sig, M


def outputs(hp, batch, graph, params, create_graph=False, ix=None):
    """(E, F, sigma, magmom, params tensor): direct heads, or with
    hp.conservative F = -dE/dr and sigma = (1/V) dE/d(eps) by autograd."""
    ix = ix or _indices(batch, graph)
    p = params if torch.is_tensor(params) else _t(params).requires_grad_(True)
    if not hp.conservative:
        E, F, sig, M = forward(hp, batch, graph, p, ix=ix)
        return E, F, sig, M, p
    pos = _t(batch.pos).requires_grad_(True)
    eps = torch.zeros((ix["S"], 3, 3), dtype=_DT, requires_grad=True)
    E, _, _, M = forward(hp, batch, graph, p, pos=pos, strain=eps, ix=ix)
    gpos, geps = torch.autograd.grad(E.sum(), (pos, eps), create_graph=create_graph)
    vol = torch.abs(torch.linalg.det(_t(batch.lattice)))
    return E, -gpos, geps / vol[:, None, None], M, p


def _pointwise(r, delta):
    if delta is None:
        return r * r
    ar = torch.abs(r)
    return torch.where(ar <= delta, 0.5 * r * r, delta * (ar - 0.5 * delta))


def loss_and_grad(hp, batch, graph, params, targets, w=(2.0, 1.5, 0.1), delta=None, w_m=0.1):
    """Training loss (prefactor-weighted means over S per-atom energies, 3N
    force components, 9S stress components, N moments) and its gradient with
    respect to the flat parameters; through F = -dE/dr with hp.conservative."""
    ix = _indices(batch, graph)
    E, F, sig, M, p = outputs(hp, batch, graph, params, create_graph=True, ix=ix)
    Et, Ft, St = (_t(x) for x in targets[:3])
    loss = (w[0] * _pointwise(E / _t(ix["n_per"]) - Et, delta).mean() + w[1] * _pointwise(F - Ft, delta).mean()
            + w[2] * _pointwise(sig - St, delta).mean())
    if hp.magmom:
        loss = loss + w_m * _pointwise(M - _t(targets[3]), delta).mean()
    (g,) = torch.autograd.grad(loss, p)
    return float(loss.detach()), g.numpy()


def numpy_outputs(hp, batch, graph, params):
    """outputs() as NumPy arrays (no gradient)."""
    with torch.enable_grad():
        E, F, sig, M, _ = outputs(hp, batch, graph, params)
    f = lambda x: None if x is None else x.detach().numpy()
    return f(E), f(F), f(sig), f(M)

