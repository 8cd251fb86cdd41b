"""Closed-form pins of the oracle's neural appearance (the paper's Sec. 4
decoder: input = (SH basis of the view direction up to the active degree,
(sin f, cos f) of each of 8 features), 32 -> 16 -> 16 -> 3 without biases,
ReLU hidden units, residual tanh(MLP(x)), colour max(0, c0 + residual + 0.5);
the residual is off while the active degree is 0). Its backward is pinned by
finite differences in test_oracle_grad.py."""
import math

import numpy as np
import pytest

from paper_2609_05255_amd import inputs

C1 = math.sqrt(3.0 / (4.0 * math.pi))


def scene(n=64):
    sc = inputs.make_scene("tiny", n=n, appearance=("neural",))
    return sc


def selector(k):
    """W1 copies input k to hidden unit 0, W2 copies unit 0, W3 copies it to all outputs."""
    w = np.zeros(816, np.float16)
    w[0 * 32 + k] = 1.0
    w[512 + 0] = 1.0
    for ch in range(3):
        w[512 + 256 + ch * 16 + 0] = 1.0
    return w.view(np.uint16)


def colours(orc, sc, cam, degree, dir_exact=True):
    pre = orc.preprocess(cam, sc, kind="neural", sh_degree=degree, mode="f64", dir_exact=dir_exact)
    vis = pre["tiles"] > 0
    assert vis.sum() > 10
    return pre["color"], vis


def directions(sc, cam):
    v = sc.means.astype(np.float64) - np.asarray(cam.campos, np.float64)[:, None]
    return v / np.linalg.norm(v, axis=0)


def base(sc):
    return sc.base_color.astype(np.float32).astype(np.float64)


def test_degree_zero_disables_the_residual(orc):
    sc = scene()
    cam = inputs.make_cameras("tiny")[0]
    col, vis = colours(orc, sc, cam, 0)
    assert np.array_equal(col[:, vis], np.maximum(0.0, base(sc) + 0.5)[:, vis])


def test_zero_output_layer_gives_the_base_colour(orc):
    sc = scene()
    w = sc.neural_w.view(np.float16).copy()
    w[768:] = 0
    sc.neural_w = w.view(np.uint16)
    cam = inputs.make_cameras("tiny")[0]
    col, vis = colours(orc, sc, cam, 3)
    assert np.array_equal(col[:, vis], np.maximum(0.0, base(sc) + 0.5)[:, vis])


@pytest.mark.parametrize("k,what", [(16, "sin f0"), (23, "cos f3"), (1, "Y1"), (4, "Y4 inactive at degree 1")])
def test_selector_networks(orc, k, what):
    sc = scene()
    sc.neural_w = selector(k)
    cam = inputs.make_cameras("tiny")[0]
    f = sc.features.view(np.float16).astype(np.float64)
    d = directions(sc, cam)
    x = {16: np.sin(f[0]), 23: np.cos(f[3]), 1: -C1 * d[1], 4: np.zeros(sc.n)}[k]
    expect = np.maximum(0.0, base(sc) + np.tanh(np.maximum(0.0, x))[None] + 0.5)
    col, vis = colours(orc, sc, cam, 1)
    assert np.allclose(col[:, vis], expect[:, vis], rtol=0, atol=1e-12), what
    # with the inputs rounded to binary16, as the half-precision decoder sees them
    col, vis = colours(orc, sc, cam, 1, dir_exact=False)
    xh = x.astype(np.float16).astype(np.float64)
    expect = np.maximum(0.0, base(sc) + np.tanh(np.maximum(0.0, xh))[None] + 0.5)
    assert np.allclose(col[:, vis], expect[:, vis], rtol=0, atol=1e-12), what


@pytest.mark.parametrize("k,degree", [(4, 2), (9, 3), (9, 2)])
def test_higher_band_inputs_follow_the_active_degree(orc, k, degree):
    # Y4 = sqrt(15/(4 pi)) x y (degree 2, m = -2; silent at degree 1, above);
    # Y9 = -sqrt(35/(32 pi)) y (3 x^2 - y^2) (degree 3, m = -3, Condon-Shortley
    # sign as band 1's -y), silent below degree 3
    sc = scene()
    sc.neural_w = selector(k)
    cam = inputs.make_cameras("tiny")[0]
    d = directions(sc, cam)
    if k == 4:
        x = math.sqrt(15.0 / (4.0 * math.pi)) * d[0] * d[1]
    else:
        x = -math.sqrt(35.0 / (32.0 * math.pi)) * d[1] * (3.0 * d[0] ** 2 - d[1] ** 2)
    if degree < (2 if k == 4 else 3):
        x = np.zeros(sc.n)
    else:
        assert (x > 0.01).sum() >= 5   # a non-trivial check: enough positive inputs
    col, vis = colours(orc, sc, cam, degree)
    expect = np.maximum(0.0, base(sc) + np.tanh(np.maximum(0.0, x))[None] + 0.5)
    assert np.allclose(col[:, vis], expect[:, vis], rtol=0, atol=1e-12)


# ---- first-layer folding (the paper's viewer; render only) ----------------------

@pytest.mark.parametrize("degree", [1, 2, 3])
def test_folding_is_exact_with_exact_inputs(orc, degree):
    # folding only regroups the first layer's sum: with exact (unrounded) inputs
    # and pre-activations the folded decoder gives the unfolded colours
    sc = scene(256)
    cam = inputs.make_cameras("tiny")[0]
    a = orc.preprocess(cam, sc, kind="neural", sh_degree=degree, mode="f64", dir_exact=True)
    b = orc.preprocess(cam, sc, kind="neural_folded", sh_degree=degree, mode="f64", dir_exact=True)
    vis = a["tiles"] > 0
    assert vis.sum() > 100 and np.array_equal(vis, b["tiles"] > 0)
    assert np.allclose(a["color"][:, vis], b["color"][:, vis], rtol=0, atol=1e-12)
    # and the residual is far from zero, so the comparison means something
    assert np.abs(a["color"][:, vis] - np.maximum(0.0, base(sc) + 0.5)[:, vis]).max() > 0.05


def test_folded_preactivations_closed_form(orc):
    # W1 row 0 = 0.75 on the constant Y_0 input and -1.5 on sin f_2; row 5 = 2 on cos f_7;
    # direction columns must not enter the pre-activations
    sc = scene(64)
    w = np.zeros(816, np.float16)
    w[0 * 32 + 0] = 0.75
    w[0 * 32 + 16 + 2 * 2] = -1.5
    w[0 * 32 + 3] = 1.0
    w[5 * 32 + 17 + 2 * 7] = 2.0
    f = sc.features.view(np.float16).astype(np.float64)
    y0 = 0.5 / math.sqrt(math.pi)
    p = orc.neural_fold(sc.features, w.view(np.uint16), exact=True)
    assert p.shape == (16, sc.n)
    assert np.allclose(p[0], 0.75 * y0 - 1.5 * np.sin(f[2]), rtol=0, atol=1e-15)
    assert np.allclose(p[5], 2.0 * np.cos(f[7]), rtol=0, atol=1e-15)
    assert not np.delete(p, [0, 5], axis=0).any()
    # stored form: binary16 inputs, the sum rounded to binary16
    h = lambda v: np.asarray(v, np.float64).astype(np.float16).astype(np.float64)
    q = orc.neural_fold(sc.features, w.view(np.uint16))
    assert np.array_equal(q[0], h(0.75 * h(y0) - 1.5 * h(np.sin(f[2]))))
    assert np.array_equal(q[5], h(2.0 * h(np.cos(f[7]))))


def test_folded_form_has_no_backward(orc):
    sc = scene(16)
    cam = inputs.make_cameras("tiny")[0]
    r = orc.render(cam, sc, kind="neural_folded", sh_degree=2, mode="f64")
    with pytest.raises(ValueError):
        orc.render_bwd(cam, sc, r["pre"], r["ranges"], r["values"], np.zeros((3, 64, 64)), kind="neural_folded")


# ---- the configurations of the paper's architecture table --------------------------

def selector_arch(layers, width, k):
    """W1 copies input k to hidden unit 0, each hidden-to-hidden layer copies unit 0,
    the output layer copies it to all three outputs."""
    w = np.zeros(32 * width + (layers - 1) * width * width + 3 * width, np.float16)
    w[k] = 1.0
    off = 32 * width
    for _ in range(layers - 1):
        w[off] = 1.0
        off += width * width
    for ch in range(3):
        w[off + ch * width] = 1.0
    return w.view(np.uint16)


@pytest.mark.parametrize("arch", [(1, 16, 0), (3, 16, 0), (2, 32, 0), (3, 32, 0), (2, 16, 1), (1, 16, 1)])
@pytest.mark.parametrize("k", [1, 16, 27])
def test_configurations_selector_networks(orc, arch, k):
    layers, width, raw16 = arch
    sc = inputs.make_scene("tiny", n=64, appearance=("neural",), neural_arch=arch)
    sc.neural_w = selector_arch(layers, width, k)
    cam = inputs.make_cameras("tiny")[0]
    f = sc.features.view(np.float16).astype(np.float64)
    d = directions(sc, cam)
    if k == 1:
        x = -C1 * d[1]
    elif raw16:
        x = f[k - 16]                       # raw features enter as they are
    else:
        j = (k - 16) // 2
        x = np.sin(f[j]) if k % 2 == 0 else np.cos(f[j])
    expect = np.maximum(0.0, base(sc) + np.tanh(np.maximum(0.0, x))[None] + 0.5)
    col, vis = colours(orc, sc, cam, 1)
    assert np.allclose(col[:, vis], expect[:, vis], rtol=0, atol=1e-12)


def routed_selector(layers, width, k):
    """Far-from-symmetric weights: W1[3][k] = 1 puts input k on hidden unit 3,
    each hidden-to-hidden matrix moves unit u to (u + 5) mod width
    (W[(u + 5) % width][u] = 1), and the output layer reads the unit the input
    ends on. Any of the matrices read in [in][out] order instead of the
    boundary's [out][in] routes another input, or none, to the outputs."""
    w = np.zeros(32 * width + (layers - 1) * width * width + 3 * width, np.float16)
    w[3 * 32 + k] = 1.0
    off, unit = 32 * width, 3
    for _ in range(layers - 1):
        for u in range(width):
            w[off + ((u + 5) % width) * width + u] = 1.0
        off += width * width
        unit = (unit + 5) % width
    for ch in range(3):
        w[off + ch * width + unit] = 1.0
    return w.view(np.uint16)


@pytest.mark.parametrize("arch", [(1, 16, 0), (2, 16, 0), (3, 16, 0), (2, 32, 0), (3, 32, 0), (2, 16, 1)])
@pytest.mark.parametrize("k", [1, 16, 27])
def test_weight_orientation(orc, arch, k):
    layers, width, raw16 = arch
    sc = inputs.make_scene("tiny", n=64, appearance=("neural",), neural_arch=arch)
    sc.neural_w = routed_selector(layers, width, k)
    cam = inputs.make_cameras("tiny")[0]
    f = sc.features.view(np.float16).astype(np.float64)
    d = directions(sc, cam)
    if k == 1:
        x = -C1 * d[1]
    elif raw16:
        x = f[k - 16]
    else:
        j = (k - 16) // 2
        x = np.sin(f[j]) if k % 2 == 0 else np.cos(f[j])
    expect = np.maximum(0.0, base(sc) + np.tanh(np.maximum(0.0, x))[None] + 0.5)
    col, vis = colours(orc, sc, cam, 1)
    assert np.allclose(col[:, vis], expect[:, vis], rtol=0, atol=1e-12)
    # the pin has teeth: the expected residual is non-zero somewhere, while a
    # transposed read of the square matrices moves the input by -5 per layer
    # (ending on a unit the output layer does not read) and a transposed
    # 32 x 32 W1 routes nothing to unit 3: either way the residual would be 0
    assert (np.maximum(0.0, x)[vis] > 0.05).any()
    if layers > 1:
        assert (3 - 5 * (layers - 1)) % width != (3 + 5 * (layers - 1)) % width


def test_configurations_weight_counts(orc):
    # the paper's default decoder has 816 parameters (Sec. 4); the table's wider
    # variant 32 -> 32 -> 32 -> 3 needs 2144 multiply-adds, all of them weights
    assert orc.neural_weight_count(2, 16) == 816
    assert orc.neural_weight_count(2, 32) == 2144
    for arch in [(1, 16, 0), (3, 16, 0), (2, 32, 0)]:
        sc = inputs.make_scene("tiny", n=8, appearance=("neural",), neural_arch=arch)
        assert sc.neural_w.size == orc.neural_weight_count(*arch[:2])
