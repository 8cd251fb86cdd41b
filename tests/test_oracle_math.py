"""Pins of the oracle's building blocks against library routines and closed forms.

SH basis (eq. sh_color_eval): scipy's complex spherical harmonics, orthonormality
by exact quadrature, Y0 = 1/sqrt(4 pi) (the SH paragraph of the appearance-model
appendix quotes 0.282), finite differences of the gradient.
binary16 rounding (the decoder runs in half precision, Sec. 4): numpy's float16.
"""
import math

import numpy as np
import pytest
import scipy.special as sp


def _real_sh_scipy(l, m, d):
    """Real SH with the Condon-Shortley phase kept: sqrt2 Re / sqrt2 Im of scipy's Y_l^|m|."""
    x, y, z = d
    theta = math.acos(max(-1.0, min(1.0, z)))
    phi = math.atan2(y, x)
    Y = sp.sph_harm_y(l, abs(m), theta, phi)
    if m == 0:
        return Y.real
    if m > 0:
        return math.sqrt(2.0) * Y.real
    return math.sqrt(2.0) * Y.imag


def _unit(v):
    v = np.asarray(v, dtype=np.float64)
    return v / np.linalg.norm(v)


def test_sh_basis_matches_scipy(orc):
    rng = np.random.default_rng(5)
    for _ in range(50):
        d = _unit(rng.standard_normal(3))
        Y, _ = orc.sh_basis(d)
        for l in range(4):
            for m in range(-l, l + 1):
                k = l * l + l + m
                assert Y[k] == pytest.approx(_real_sh_scipy(l, m, d), abs=1e-13)


def test_sh_band0_and_band1_closed_forms(orc):
    # Y0 = 1/sqrt(4 pi) ~= 0.282; band 1 = sqrt(3/(4 pi)) * (-y, z, -x)
    d = _unit([0.3, -0.5, 0.8])
    Y, _ = orc.sh_basis(d)
    assert Y[0] == pytest.approx(1.0 / math.sqrt(4 * math.pi), rel=1e-15)
    assert round(Y[0], 3) == 0.282
    c1 = math.sqrt(3.0 / (4 * math.pi))
    assert Y[1:4] == pytest.approx([-c1 * d[1], c1 * d[2], -c1 * d[0]], rel=1e-14)


def test_sh_orthonormal_by_quadrature(orc):
    # Gauss-Legendre in z (exact to degree 2*8-1) x uniform in phi (exact for |m| < 16)
    zs, wz = np.polynomial.legendre.leggauss(8)
    nphi = 16
    G = np.zeros((16, 16))
    for z, w in zip(zs, wz):
        s = math.sqrt(1 - z * z)
        for j in range(nphi):
            phi = 2 * math.pi * j / nphi
            Y, _ = orc.sh_basis([s * math.cos(phi), s * math.sin(phi), z])
            G += np.outer(Y, Y) * w * (2 * math.pi / nphi)
    assert np.allclose(G, np.eye(16), atol=1e-13)


def test_sh_gradient_finite_difference(orc):
    rng = np.random.default_rng(6)
    h = 1e-6
    for _ in range(20):
        d = rng.standard_normal(3)
        _, dY = orc.sh_basis(d)
        for j in range(3):
            e = np.zeros(3)
            e[j] = h
            fd = (orc.sh_basis(d + e)[0] - orc.sh_basis(d - e)[0]) / (2 * h)
            assert np.allclose(dY[:, j], fd, atol=1e-7 * max(1.0, np.abs(fd).max()))


def test_round_half_matches_numpy(orc):
    rng = np.random.default_rng(7)
    vals = np.concatenate([
        rng.standard_normal(2000) * 0.5,
        rng.standard_normal(500) * 1e-5,           # subnormal range of binary16
        rng.standard_normal(200) * 3e4,
        np.array([0.0, -0.0, 65504.0, 65519.0, 65520.0, 1e-8, 6.1e-5, 2.0 ** -25, 3 * 2.0 ** -26]),
        # exact ties between binary16 neighbours (round half to even)
        (np.arange(1, 200) + 0.5) * 2.0 ** -10,
    ])
    for v in vals:
        expect = float(np.float64(v).astype(np.float16))
        got = orc.round_half(float(v))
        assert (got == expect) or (math.isinf(got) and math.isinf(expect) and got == expect), (v, got, expect)


def test_paper_printed_values(orc):
    """Values printed in the paper (tests/golden/paper_printed_values.json)."""
    import json
    import os
    with open(os.path.join(os.path.dirname(__file__), "golden", "paper_printed_values.json")) as f:
        gold = json.load(f)
    d = np.array([0.3, -0.5, 0.8])
    y, _ = orc.sh_basis(d / np.linalg.norm(d))
    g = gold["sh_y0"]
    assert round(float(y[0]), g["decimals"]) == g["value"]
    # degree-3 SH: 16 basis functions per colour channel, fp32
    assert len(y) * 3 * 4 == gold["sh3_appearance_bytes"]["value"]
    from paper_2609_05255_amd import inputs
    sc = inputs.make_scene("tiny", n=8, appearance=("latent",))
    assert sc.latent.shape[0] * sc.latent.dtype.itemsize == gold["latent_appearance_bytes_measured_decoder"]["value"]
    # the neural model and its configurations
    assert orc.neural_weight_count(2, 16) == gold["neural_decoder_parameters"]["value"]
    assert orc.neural_weight_count(2, 32) == gold["neural_32_wide_macs"]["value"]
    sc = inputs.make_scene("tiny", n=8, appearance=("neural",))
    per_g = lambda *arrays: sum(a.shape[0] * a.dtype.itemsize for a in arrays)
    assert per_g(sc.base_color, sc.features) == gold["neural_appearance_bytes"]["value"]
    sc = inputs.make_scene("tiny", n=8, appearance=("neural",), neural_arch=(2, 16, 1))
    assert per_g(sc.base_color, sc.features) == gold["neural_f16_bytes"]["value"]
    sc = inputs.make_scene("tiny", n=8, appearance=("nasg", "nasgabor"))
    assert per_g(sc.base_color, sc.lobes) == gold["nasg_appearance_bytes"]["value"]
    assert per_g(sc.base_color, sc.lobes_gabor) == gold["nasgabor_appearance_bytes"]["value"]
