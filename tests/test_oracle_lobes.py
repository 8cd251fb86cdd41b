"""Pins of the oracle's NASG and NASGabor lobe (eq. nasg; the kernel of Huang
et al.'s normalized anisotropic spherical Gaussian with the activations the
paper describes: tanh-mapped frame angles, clamped-exp sharpness and
anisotropy, a 20 (tanh + 1) Gabor frequency). The frame is checked against
scipy's ZYZ Euler rotation, the kernel against its closed forms along the
frame axes and its unit integral over the sphere, the derivatives against
central differences, and the appearance against its definition."""
import math

import numpy as np
import pytest
from scipy.spatial.transform import Rotation

from paper_2609_05255_amd import inputs

RAWS = [[0.3, -0.4, 0.9, 1.0, -0.5, 0.2], [1.5, 2.0, -1.0, 2.5, 1.2, -1.0], [-0.7, 0.1, 0.2, -1.0, -3.0, 0.5],
        [0.0, 0.0, 0.0, 3.0, 0.0, -2.0], [-2.0, -1.2, 1.7, 0.4, 1.9, 1.5]]


def frame(raw):
    """(x, y, z) axes: ZYZ Euler angles phi, theta, gamma with cos theta = tanh r0
    and the half angles of phi and gamma of cosine tanh r1, tanh r2."""
    th = math.acos(math.tanh(raw[0]))
    ph = 2.0 * math.acos(math.tanh(raw[1]))
    ga = 2.0 * math.acos(math.tanh(raw[2]))
    R = Rotation.from_euler("ZYZ", [ph, th, ga]).as_matrix()
    return R[:, 0], R[:, 1], R[:, 2]


def shape(raw):
    lam = math.exp(min(max(raw[3], -8.0), 8.0))
    a = math.exp(min(max(raw[4], -8.0), 8.0))
    K = 2.0 * math.pi * (1.0 - math.exp(-2.0 * lam)) / (lam * math.sqrt(1.0 + a))
    return lam, a, K


def sphere_quadrature(nz=400, nphi=800):
    z, w = np.polynomial.legendre.leggauss(nz)
    phi = (np.arange(nphi) + 0.5) * 2.0 * np.pi / nphi
    Z = np.repeat(z, nphi)
    P = np.tile(phi, nz)
    s = np.sqrt(1.0 - Z * Z)
    return np.stack([s * np.cos(P), s * np.sin(P), Z], 1), np.repeat(w, nphi) * 2.0 * np.pi / nphi


@pytest.mark.parametrize("raw", RAWS)
def test_nasg_integrates_to_one(orc, raw):
    # the normalization K makes every lobe a density on the sphere
    v, w = sphere_quadrature()
    total = float((orc.lobe_eval(raw[:5], False, v) * w).sum())
    assert abs(total - 1.0) < 2e-6, total


@pytest.mark.parametrize("raw", RAWS)
def test_nasg_along_its_frame_axes(orc, raw):
    x, y, z = frame(raw)
    lam, a, K = shape(raw)
    # the peak at z: 1/K
    assert math.isclose(orc.lobe_eval(raw[:5], False, z[None])[0], 1.0 / K, rel_tol=1e-12)
    for t in (0.3, 1.1, 2.4):
        u = (math.cos(t) + 1.0) / 2.0
        # towards x the full anisotropy applies (psi = a) ...
        gx = math.exp(2.0 * lam * (u ** (1.0 + a) - 1.0)) * u ** a / K
        # ... towards y none (psi = 0): the isotropic spherical Gaussian exp(lambda (cos t - 1)) / K
        gy = math.exp(lam * (math.cos(t) - 1.0)) / K
        vx = math.cos(t) * z + math.sin(t) * x
        vy = math.cos(t) * z + math.sin(t) * y
        got = orc.lobe_eval(raw[:5], False, np.stack([vx, vy]))
        assert math.isclose(got[0], gx, rel_tol=1e-11, abs_tol=1e-300)
        assert math.isclose(got[1], gy, rel_tol=1e-11, abs_tol=1e-300)


@pytest.mark.parametrize("raw", RAWS)
def test_nasgabor_carrier(orc, raw):
    x, y, z = frame(raw)
    omega = 20.0 * (math.tanh(raw[5]) + 1.0)
    rng = np.random.default_rng(3)
    v = rng.standard_normal((50, 3))
    v /= np.linalg.norm(v, axis=1, keepdims=True)
    base = orc.lobe_eval(raw[:5], False, v)
    got = orc.lobe_eval(raw, True, v)
    expect = base * (1.0 + np.cos(omega * (v @ x))) / 2.0
    assert np.allclose(got, expect, rtol=1e-12, atol=0)


def test_clamped_shape_parameters(orc):
    v = np.array([[0.6, 0.0, 0.8], [0.0, -0.6, 0.8]])
    a = orc.lobe_eval([0.1, 0.2, 0.3, 8.0, -8.0], False, v)
    b = orc.lobe_eval([0.1, 0.2, 0.3, 11.0, -12.0], False, v)
    assert np.array_equal(a, b)
    _, dr, _ = orc.lobe_grad([0.1, 0.2, 0.3, 11.0, -12.0], False, v[0])
    assert dr[3] == 0.0 and dr[4] == 0.0


@pytest.mark.parametrize("gabor", [False, True])
@pytest.mark.parametrize("raw", RAWS)
def test_lobe_derivatives_by_central_differences(orc, raw, gabor):
    raw = np.array(raw[: 6 if gabor else 5])
    rng = np.random.default_rng(int(abs(raw[0]) * 100) + gabor)
    for _ in range(4):
        v = rng.standard_normal(3)
        v /= np.linalg.norm(v)
        G, dr, dv = orc.lobe_grad(raw, gabor, v)
        assert math.isclose(G, orc.lobe_eval(raw, gabor, v[None])[0], rel_tol=1e-14)
        h = 1e-6
        for k in range(raw.size):
            e = np.zeros(raw.size)
            e[k] = h
            fd = (orc.lobe_eval(raw + e, gabor, v[None])[0] - orc.lobe_eval(raw - e, gabor, v[None])[0]) / (2 * h)
            assert abs(fd - dr[k]) <= 1e-6 * (abs(fd) + G + 1e-3), (k, fd, dr[k])
        for j in range(3):
            e = np.zeros(3)
            e[j] = h
            fd = (orc.lobe_eval(raw, gabor, (v + e)[None])[0] - orc.lobe_eval(raw, gabor, (v - e)[None])[0]) / (2 * h)
            assert abs(fd - dv[j]) <= 1e-6 * (abs(fd) + G + 1e-3), (j, fd, dv[j])


@pytest.mark.parametrize("kind", ["nasg", "nasgabor"])
def test_lobe_appearance(orc, kind):
    sc = inputs.make_scene("tiny", n=128, appearance=(kind,))
    cam = inputs.make_cameras("tiny")[0]
    lobes = (sc.lobes_gabor if kind == "nasgabor" else sc.lobes).astype(np.float64)
    c0 = sc.base_color.astype(np.float64)
    pre = orc.preprocess(cam, sc, kind=kind, sh_degree=1, mode="f64")
    vis = pre["tiles"] > 0
    assert vis.sum() > 30
    v = sc.means.astype(np.float64) - np.asarray(cam.campos, np.float64)[:, None]
    v /= np.linalg.norm(v, axis=0)
    for i in np.nonzero(vis)[0]:
        raw = np.concatenate([lobes[:5, i], lobes[8:9, i]]) if kind == "nasgabor" else lobes[:5, i]
        G = orc.lobe_eval(raw, kind == "nasgabor", v[:, i][None])[0]
        expect = np.maximum(0.0, c0[:, i] + G * np.tanh(lobes[5:8, i]) + 0.5)
        assert np.allclose(pre["color"][:, i], expect, rtol=0, atol=1e-13)
    # degree 0: the lobe is not yet active
    pre0 = orc.preprocess(cam, sc, kind=kind, sh_degree=0, mode="f64")
    assert np.array_equal(pre0["color"][:, vis], np.maximum(0.0, c0 + 0.5)[:, vis])
