"""Pins of the oracle's basis functions against closed forms and textbook
special functions (sRBF of Eq. (2) with the envelope reading of Eq. (12)-(13),
and the Fourier angular basis)."""
import math

import numpy as np
from scipy import integrate, special

from oracle import model


def test_envelope_from_its_derivative():
    """u(0)=1 and u'(x) = -(p(p+1)(p+2)/2) x^(p-1) (1-x)^2 (so u, u', u''
    vanish at 1); integrate the derivative and compare."""
    for p in (5, 6, 8):
        k = p * (p + 1) * (p + 2) / 2.0
        for x in np.linspace(0.0, 1.0, 11):
            integral, _ = integrate.quad(lambda t: t ** (p - 1) * (1 - t) ** 2, 0.0, x, epsabs=1e-14)
            assert abs(model.envelope(x, p) - (1.0 - k * integral)) < 1e-12
        assert model.envelope(0.0, p) == 1.0
        assert abs(model.envelope(1.0, p)) < 1e-12
        # the printed Eq. (12) coefficient p(p+2)/2 would give u(1) = -4 at p = 8
    assert abs(1 - 45 + 80 - 36 * 1.0) < 1e-12  # p = 8: 1 - 45 x^8 + 80 x^9 - 36 x^10 at x = 1


def test_srbf_is_spherical_bessel_j0():
    c, p = 6.0, 8
    r = np.linspace(0.3, 5.99, 57)
    f = np.pi * np.arange(1, 32)
    got = model.srbf(r, f, c, p)
    for n in range(1, 32):
        x = n * np.pi * r / c
        want = math.sqrt(2.0 / c) * (n * np.pi / c) * special.spherical_jn(0, x) * model.envelope(r / c, p)
        np.testing.assert_allclose(got[:, n - 1], want, rtol=1e-12, atol=1e-14)


def test_srbf_frequency_derivative():
    c, p = 3.0, 8
    r = np.linspace(0.5, 2.9, 13)
    f = np.pi * np.arange(1, 8) + 0.1 * np.sin(np.arange(7))
    h = 1e-6
    fd = (model.srbf(r, f + h, c, p) - model.srbf(r, f - h, c, p)) / (2 * h)
    np.testing.assert_allclose(model.srbf_dfreq(r, f, c, p), fd, rtol=1e-7, atol=1e-9)


def test_fourier_orthonormal_and_special_values():
    K = 31
    th = np.linspace(-np.pi, np.pi, 4096, endpoint=False)
    F = model.fourier(th, K)
    gram = F.T @ F * (2 * np.pi / th.size)  # exact for trigonometric polynomials
    np.testing.assert_allclose(gram, np.eye(K), atol=1e-12)
    v = model.fourier(np.array([np.pi / 2, np.pi]), K)
    m = np.arange(1, 16)
    np.testing.assert_allclose(v[0, 1:16] * math.sqrt(math.pi), np.cos(m * np.pi / 2), atol=1e-12)
    np.testing.assert_allclose(v[0, 16:] * math.sqrt(math.pi), [[0, 1, 0, -1][k % 4] for k in m], atol=1e-12)
    np.testing.assert_allclose(v[1, 1:16] * math.sqrt(math.pi), (-1.0) ** m, atol=1e-12)
    np.testing.assert_allclose(v[1, 16:], 0.0, atol=1e-12)
    assert abs(v[0, 0] - 1 / math.sqrt(2 * math.pi)) < 1e-15


def test_angle_matches_arccos_definition():
    """theta_ijk = arccos(r_ij . r_ik / (|r_ij| |r_ik|)) (Sec. II-B (1)); the
    oracle evaluates it as atan2(|a x b|, a . b)."""
    from oracle import graph
    from paper_2412_20796_amd import synth

    b = synth.random_crystals(seed=11, n_struct=2, n_lo=6, n_hi=10)
    g = graph.build_graph(b.atom_ptr, b.pos, b.lattice)
    dv = model.derived(b, g)
    ra = dv["rvec"][dv["bond_edge"][dv["b1"]]]
    rb = dv["rvec"][dv["bond_edge"][dv["b2"]]]
    cosv = (ra * rb).sum(1) / np.linalg.norm(ra, axis=1) / np.linalg.norm(rb, axis=1)
    ok = np.abs(cosv) < 0.999
    assert ok.sum() > 10
    np.testing.assert_allclose(dv["theta"][ok], np.arccos(cosv[ok]), atol=1e-10)
