"""GPU parity of the HIP path (through the C ABI) with the CPU oracle.

Bit-exact: culling, tiles touched, tile rectangles, depth keys, the projected
means/conics/opacities (one correctly rounded fp32 operation sequence on both
sides), the number of pairs, the sorted per-tile lists, tile ids and ranges.
Images: abs 1e-5 + rel 1e-4 on every pixel whose decisions lie outside the
rounding bound of the oracle's margin; the others (flagged) are counted and
bounded, and get a zero upstream gradient on both sides.
Gradients (the fp32 tolerance of the workload): every element within 1e-3 |ref| + 1e-5 max|ref|
and relative L2 <= 1e-4 per tensor; the decoder paths as stated in MLP_GRADS.
"""
import numpy as np
import pytest

from paper_2609_05255_amd import inputs

import torch

from oracle import oracle as orc
from paper_2609_05255_amd import gsraster as gs
from parity import (MLP_ATOL, MLP_HALF_ATOL, MLP_GRADS, NEURAL_FLIP, check_grads, compare_image, compare_lists,
                    compare_preprocess, flagged_pixels, grad_stats, lobe_color_atol, report_grads, run_gpu, say,
                    tiny_camera)

pytestmark = pytest.mark.gpu


def check_all(scene, cam, kind="sh3", sh_degree=3, label="", grads=True, capacity=None, max_flagged=None,
              cam_seed=0):
    say("case %s: n=%d %dx%d %s degree %d" % (label, scene.n, cam.width, cam.height, kind, sh_degree))
    latent = kind in ("latent", "neural", "neural_folded")
    # the decoder's operands are binary16: compare with the oracle that rounds them alike
    ref = orc.render(cam, scene, kind=kind, sh_degree=sh_degree, mode="f32", half_act=latent)
    flagged = flagged_pixels(ref["margin"], max_flagged)
    g = None
    if grads:
        g = (inputs.make_upstream_grad(cam.width, cam.height, cam_seed) * ~flagged[None]).astype(np.float32)
        ref["grads"] = orc.render_bwd(cam, scene, ref["pre"], ref["ranges"], ref["values"], g, kind=kind,
                                      sh_degree=sh_degree, mode="f32", half_act=latent)
    gpu = run_gpu(scene, cam, kind, sh_degree, g, capacity=capacity)
    flip = NEURAL_FLIP if kind in ("neural", "neural_folded") else None
    atol = (MLP_HALF_ATOL if latent else
            lobe_color_atol(scene, cam, kind, ref["pre"]["color"], sh_degree) if kind in ("nasg", "nasgabor") else 2e-6)
    compare_preprocess(gpu, ref["pre"], color_atol=atol, flip=flip)
    compare_lists(gpu, ref["values"], ref["tile_of"], ref["ranges"])
    if latent:
        compare_image(gpu, ref["image"], ref["final_T"], ref["n_contrib"], ref["margin"],
                      atol=flip[0] if flip else MLP_HALF_ATOL, rtol=0.0)
        exact = orc.render(cam, scene, kind=kind, sh_degree=sh_degree, mode="f32")
        err = np.abs(gpu["image"] - exact["image"])[:, exact["margin"] > 1.0]
        say("  latent image vs the exact decoder: max abs %.2e" % (err.max() if err.size else 0.0))
        assert err.size == 0 or err.max() <= MLP_ATOL
    else:
        compare_image(gpu, ref["image"], ref["final_T"], ref["n_contrib"], ref["margin"])
    say("  P=%d" % gpu["P"])
    if grads:
        st = grad_stats(gpu["grads"], ref["grads"])
        report_grads(st)
        if kind in ("latent", "neural"):
            check_grads(st, **MLP_GRADS)
        else:
            check_grads(st)
    return gpu, ref


def test_tiny_scene():
    sc = inputs.make_scene("tiny")
    cam = inputs.make_cameras("tiny")[0]
    check_all(sc, cam, label="tiny", max_flagged=0)


@pytest.mark.parametrize("degree", [0, 1, 2])
def test_tiny_scene_lower_sh_degrees(degree):
    sc = inputs.make_scene("tiny")
    check_all(sc, inputs.make_cameras("tiny")[0], sh_degree=degree, label="tiny", max_flagged=0)


def test_ragged_image_with_background():
    # 50x37 pixels: partial edge tiles on both axes; non-black background
    sc = inputs.make_scene("tiny")
    check_all(sc, tiny_camera(50, 37, bg=(0.25, 0.5, 0.75)), label="ragged")


@pytest.mark.parametrize("size", [(16, 16), (17, 9), (300, 20)])
def test_tile_grid_edge_cases(size):
    # one tile (no tile-sort pass), two tiles, and a 19x2 grid
    sc = inputs.make_scene("tiny")
    check_all(sc, tiny_camera(*size), label="grid%dx%d" % size)


def test_more_than_65536_tiles():
    # 4097 x 16 tiles: the tile ids no longer fit 16 bits, so the pair emission
    # and the tile sort carry 32-bit keys (below that they carry 16-bit ones)
    sc = inputs.make_scene("tiny").subset(np.arange(300))
    check_all(sc, tiny_camera(16 * 4097, 256), label="wide", grads=False)


@pytest.mark.parametrize("tiles_x", [2048, 2049])
def test_backward_tile_order_limit(tiles_x):
    # 2048 x 16 = 32768 tiles, the largest image whose backward launches its
    # tiles longest walk first (as every other case here), and 2049 x 16, the
    # smallest that keeps the plain tile order
    sc = inputs.make_scene("tiny").subset(np.arange(300))
    check_all(sc, tiny_camera(16 * tiles_x, 256), label="wide-bwd-%d" % tiles_x)


@pytest.mark.parametrize("degree", [3, 1])
def test_sh3_backward_without_the_colour_jacobian(degree):
    # gs_preprocessed.color_jac NULL: the preprocess writes no view-direction
    # Jacobian and the backward re-reads the SH coefficients instead. The same
    # gradients as with it (the oracle checks the Jacobian path in every other
    # SH3 case), to the float atomics' summation order and a few ulp of the two
    # evaluation orders of the direction term.
    sc = inputs.make_scene("medium")
    cam = inputs.make_cameras("medium")[6]
    say("case SH3 backward from the coefficients, degree %d" % degree)
    up = torch.from_numpy(inputs.make_upstream_grad(cam.width, cam.height, 6)).cuda()
    st = gs.SceneTensors(sc)
    cs = gs.camera_struct(cam)
    out = []
    for jac in (True, False):
        fr = gs.Frame(sc.n, cam.width, cam.height, gs.GS_APP_SH3, 1 << 22)
        if not jac:
            fr.pre.color_jac = None
        fr.forward(cs, st, degree)
        fr.backward(cs, st, up, degree)
        torch.cuda.synchronize()
        out.append({k: getattr(fr, k).clone() for k in ("dmeans", "dlog_scales", "dquats", "dopacity_logits", "dsh")})
        out[-1]["image"] = fr.image.clone()
    assert torch.equal(out[0]["image"], out[1]["image"])
    for k in ("dmeans", "dlog_scales", "dquats", "dopacity_logits", "dsh"):
        a, b = out[0][k], out[1][k]
        scale = float(b.abs().max())
        err = float((a - b).abs().max())
        say("  %s: max |diff| %.2e of max |grad| %.2e" % (k, err, scale))
        assert bool(((a - b).abs() <= 1e-4 * b.abs() + 1e-6 * scale).all()), k


def test_capacity_retry():
    sc = inputs.make_scene("tiny")
    check_all(sc, inputs.make_cameras("tiny")[0], capacity=100, label="capacity")


def test_empty_and_culled_scenes():
    sc = inputs.make_scene("tiny")
    empty = sc.subset(np.arange(0))
    gpu, ref = check_all(empty, tiny_camera(40, 24, bg=(0.3, 0.6, 0.9)), label="empty")
    assert np.all(gpu["image"][0] == np.float32(0.3))
    # camera looking away from every Gaussian
    away = inputs.look_at_camera([0.0, 0.0, -3.0], 64, 64, target=(0.0, 0.0, -6.0))
    gpu, ref = check_all(sc, away, label="culled")
    assert gpu["P"] == 0 and np.all(gpu["tiles"] == 0)
    for k, v in gpu["grads"].items():
        assert np.all(v == 0), k


@pytest.mark.parametrize("cam_index", range(8))
def test_medium_scene(cam_index):
    # every camera of the medium workload (200k Gaussians, 1280x720)
    sc = inputs.make_scene("medium")
    check_all(sc, inputs.make_cameras("medium")[cam_index], label="medium cam %d" % cam_index, cam_seed=cam_index)


def test_mlp_eval_matches_oracle():
    rng = np.random.default_rng(31)
    rows = 1000                                 # 15 full waves and a ragged one
    x = rng.normal(0.0, 0.5, size=(rows, 17))
    x[:, 14:] /= np.linalg.norm(x[:, 14:], axis=1, keepdims=True)
    x[7] = 0.0                                  # all-zero input: every hidden unit at 0
    xb = x.astype(np.float16).view(np.uint16)
    w = inputs.make_mlp_weights(5)
    say("case mlp_eval rows=%d" % rows)
    xt = torch.from_numpy(xb.view(np.int16)).cuda()
    wt = torch.from_numpy(w.view(np.int16)).cuda()
    out = torch.empty(rows, 3, device="cuda")
    gs.gs_mlp_eval(xt, rows, wt, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    err = np.abs(got - orc.mlp_eval(xb, w))
    err_half = np.abs(got - orc.mlp_eval(xb, w, half_act=True))
    say("  max abs error %.2e (exact decoder), %.2e (binary16 activations)" % (err.max(), err_half.max()))
    assert err.max() <= MLP_ATOL
    assert err_half.max() <= MLP_HALF_ATOL
    assert np.all(got[7] == 0.5)


def test_tiny_scene_latent():
    sc = inputs.make_scene("tiny", appearance=("latent",))
    check_all(sc, inputs.make_cameras("tiny")[0], kind="latent", label="tiny latent", max_flagged=0)


def test_ragged_latent_with_background():
    sc = inputs.make_scene("tiny", appearance=("latent",))
    check_all(sc, tiny_camera(50, 37, bg=(0.25, 0.5, 0.75)), kind="latent", label="ragged latent")


@pytest.mark.parametrize("cam_index", [2, 6])
def test_medium_scene_latent(cam_index):
    sc = inputs.make_scene("medium", appearance=("latent",))
    check_all(sc, inputs.make_cameras("medium")[cam_index], kind="latent", label="medium latent cam %d" % cam_index,
              cam_seed=cam_index)


@pytest.mark.parametrize("degree", [0, 1, 2, 3])
def test_tiny_scene_neural(degree):
    # the paper's neural appearance; degree 0 has the residual off
    sc = inputs.make_scene("tiny", appearance=("neural",))
    check_all(sc, tiny_camera(), kind="neural", sh_degree=degree, label="tiny-neural", max_flagged=0)


def test_ragged_neural_with_background():
    sc = inputs.make_scene("tiny", appearance=("neural",))
    check_all(sc, tiny_camera(50, 37, bg=(0.1, 0.5, 0.9)), kind="neural", label="ragged-neural")


def test_medium_scene_neural():
    sc = inputs.make_scene("medium", appearance=("neural",))
    check_all(sc, inputs.make_cameras("medium")[2], kind="neural", label="medium-neural")


def test_binning_one_tile_and_huge_gaussians():
    # 6000 Gaussians so small that nearly all touch one tile (a window of 64
    # consecutive pairs then holds up to 64 Gaussians), plus a few so large
    # they cover the whole 96x80 image; pairs span several emission chunks
    import dataclasses
    # (the scene's own anisotropic log-scales, shifted: with equal axes the
    # covariance would not depend on the rotation and the exact quaternion
    # gradient would be zero, leaving only rounding to compare)
    sc = inputs.make_scene("tiny", n=6000)
    ls = (sc.log_scales - np.float32(3.5)).astype(np.float32)
    ls[:, ::997] += np.float32(6.0)
    sc = dataclasses.replace(sc, log_scales=ls)
    check_all(sc, tiny_camera(96, 80), label="one-tile+huge")


# ---- the folded neural form (render only) ---------------------------------------

def folded_preact_check(sc, got):
    """GPU pre-activations against the oracle's fold (binary16 inputs, fp64 sum,
    rounded to binary16). The GPU's sin/cos (fp32) may round an input to the
    neighbouring binary16 value (spacing <= 2^-11 below 1), which moves a sum
    by at most max|W1| 2^-11, and it sums in fp32 (17 terms, error far below
    1e-5); the final rounding then adds at most one binary16 spacing. Both are
    rare: nearly every value is bit-equal."""
    ref = orc.neural_fold(sc.features, sc.neural_w).T          # [n][16]
    g = got.view(np.float16).astype(np.float64)
    assert g.shape == ref.shape
    w1 = np.abs(sc.neural_w.view(np.float16).astype(np.float64)[:512])
    spacing = np.spacing(np.abs(ref).astype(np.float16)).astype(np.float64)
    diff = np.abs(g - ref)
    bound = spacing + w1.max() * 2.0 ** -11 + 1e-5
    assert np.all(diff <= bound), float((diff / bound).max())
    flips = int((diff > 0).sum())
    say("  fold: %d of %d pre-activations on the neighbouring binary16 value" % (flips, ref.size))
    assert flips <= max(2, ref.size // 1000)


@pytest.mark.parametrize("n", [1, 63, 1000, 4096])
def test_neural_fold(n):
    sc = inputs.make_scene("tiny", n=n, appearance=("neural",))
    st = gs.SceneTensors(sc)
    got = st.fold_neural().cpu().numpy().view(np.uint16)
    torch.cuda.synchronize()
    folded_preact_check(sc, got)


def test_neural_fold_empty():
    sc = inputs.make_scene("tiny", n=1, appearance=("neural",))
    st = gs.SceneTensors(sc)
    st.preact = torch.full((1, 16), 7, dtype=torch.int16, device="cuda")
    gs.gs_neural_fold(st.features, st.neural_w, 0, st.preact)   # n = 0 touches nothing
    torch.cuda.synchronize()
    assert np.all(st.preact.cpu().numpy() == 7)


@pytest.mark.parametrize("degree", [0, 1, 2, 3])
def test_tiny_scene_neural_folded(degree):
    sc = inputs.make_scene("tiny", appearance=("neural",))
    check_all(sc, tiny_camera(), kind="neural_folded", sh_degree=degree, label="tiny-folded", grads=False)


def test_ragged_neural_folded_with_background():
    sc = inputs.make_scene("tiny", n=1000, appearance=("neural",))
    check_all(sc, tiny_camera(50, 37, bg=(0.3, 0.2, 0.1)), kind="neural_folded", label="ragged-folded",
              grads=False)


def test_medium_scene_neural_folded():
    sc = inputs.make_scene("medium", appearance=("neural",))
    check_all(sc, inputs.make_cameras("medium")[2], kind="neural_folded", label="medium-folded", grads=False)


# ---- NASG and NASGabor lobes ------------------------------------------------------

@pytest.mark.parametrize("kind", ["nasg", "nasgabor"])
@pytest.mark.parametrize("degree", [0, 1])
def test_tiny_scene_lobe(kind, degree):
    sc = inputs.make_scene("tiny", appearance=(kind,))
    check_all(sc, tiny_camera(), kind=kind, sh_degree=degree, label="tiny-" + kind)


@pytest.mark.parametrize("kind", ["nasg", "nasgabor"])
def test_ragged_lobe_with_background(kind):
    sc = inputs.make_scene("tiny", n=999, appearance=(kind,))
    check_all(sc, tiny_camera(50, 37, bg=(0.6, 0.1, 0.4)), kind=kind, label="ragged-" + kind)


@pytest.mark.parametrize("kind", ["nasg", "nasgabor"])
def test_medium_scene_lobe(kind):
    sc = inputs.make_scene("medium", appearance=(kind,))
    check_all(sc, inputs.make_cameras("medium")[5], kind=kind, label="medium-" + kind)


@pytest.mark.parametrize("degree", [0, 3])
def test_tiny_scene_sh_y0_folded(degree):
    # the paper's implementation: DC coefficients stored with Y0 folded in
    sc = inputs.make_scene("tiny")
    sc.sh = sc.sh.copy()
    sc.sh[0:3] *= np.float32(0.28209479177387814)
    sc.sh_y0_folded = True
    check_all(sc, tiny_camera(), sh_degree=degree, label="tiny-sh-y0-folded")


# ---- the neural decoder configurations of the paper's architecture table ---------

@pytest.mark.parametrize("arch", [(1, 16, 0), (3, 16, 0), (2, 16, 1), (3, 16, 1), (2, 32, 0)])
def test_tiny_scene_neural_configurations(arch):
    sc = inputs.make_scene("tiny", appearance=("neural",), neural_arch=arch)
    check_all(sc, tiny_camera(), kind="neural", sh_degree=3, label="tiny-neural-%d-%d-%d" % arch)


@pytest.mark.parametrize("degree", [0, 1, 2])
def test_tiny_scene_neural_32_wide_degrees(degree):
    # degree masking of the direction inputs (degree 0: the residual is off)
    sc = inputs.make_scene("tiny", appearance=("neural",), neural_arch=(2, 32, 0))
    check_all(sc, tiny_camera(), kind="neural", sh_degree=degree, label="tiny-neural-2-32-0")


def test_ragged_neural_32_wide_with_background():
    sc = inputs.make_scene("tiny", appearance=("neural",), neural_arch=(2, 32, 0))
    check_all(sc, tiny_camera(50, 37, bg=(0.1, 0.5, 0.9)), kind="neural", label="ragged-neural-2-32-0")


def test_medium_scene_neural_32_wide():
    sc = inputs.make_scene("medium", appearance=("neural",), neural_arch=(2, 32, 0))
    check_all(sc, inputs.make_cameras("medium")[2], kind="neural", label="medium-neural-2-32-0")


def test_medium_scene_neural_three_layers():
    sc = inputs.make_scene("medium", appearance=("neural",), neural_arch=(3, 16, 0))
    check_all(sc, inputs.make_cameras("medium")[2], kind="neural", label="medium-neural-3-16-0")


# ---- degenerate Gaussians ----------------------------------------------------------

def degenerate_scene():
    """The tiny scene with extreme members: needle-thin and screen-sized scales,
    opacities at the alpha cap and far below 1/255, means behind the camera,
    just beyond the near plane, on tile and pixel boundaries, and one Gaussian
    that projects far outside the image (guard band)."""
    sc = inputs.make_scene("tiny")
    f32 = np.float32
    m, ls, lg = sc.means, sc.log_scales, sc.opacity_logits
    ls[:, 0:20] = f32(-12.0)                   # far below a pixel
    ls[:, 20:30] = f32(0.5)                    # covering the whole image
    ls[0, 30:40] = f32(-1.0)                   # needles: one long axis
    ls[1:, 30:40] = f32(-9.0)
    lg[40:60] = f32(25.0)                      # opacity 1 -> alpha capped at 0.99
    lg[60:80] = f32(-25.0)                     # opacity ~ 1e-11, never 1/255
    m[:, 80:90] = np.array([[0.1], [0.2], [-3.5]], f32)          # behind the camera (it sits at z = -3)
    m[:, 90:100] = np.array([[0.0], [0.0], [-2.8 + 1e-4]], f32)  # just beyond the near plane 0.2
    cam = tiny_camera()
    # means whose projections land on tile corners and pixel centres
    fx = cam.fx
    for k, (u, v) in enumerate([(16, 16), (32, 48), (0.5, 0.5), (63.5, 31.5), (48, 0)]):
        # at depth 3 (z = 0 in the world) these land on tile corners and pixel
        # centres (the camera's x axis points along world -x, so u is mirrored)
        m[:, 100 + k] = np.array([(u - cam.cx) * 3.0 / fx, (v - cam.cy) * 3.0 / fx, 0.0], f32)
    m[:, 110] = np.array([3.0, 0.0, 0.0], f32)   # projects far to the side
    ls[:, 110] = f32(-0.5)
    return sc, cam


@pytest.mark.parametrize("kind", ["sh3", "neural", "nasg"])
def test_degenerate_gaussians(kind):
    sc, cam = degenerate_scene()
    if kind != "sh3":
        extra = inputs.make_scene("tiny", appearance=(kind,))
        sc.base_color = extra.base_color
        sc.features, sc.neural_w, sc.lobes, sc.lobes_gabor = (extra.features, extra.neural_w, extra.lobes,
                                                              extra.lobes_gabor)
    check_all(sc, cam, kind=kind, label="degenerate-" + kind)


# ---- the pair count read on the device -------------------------------------------

@pytest.mark.parametrize("size", [(64, 64), (16, 16)])
def test_device_pair_count(size):
    # gs_bin_sort in device mode (no read-back of P): the same lists, ranges and
    # image as the host mode; with a capacity below P nothing is listed, every
    # range is empty, the image is the background, the gradients are zero, and
    # pre->num_pairs keeps the P needed for the retry
    sc = inputs.make_scene("tiny")
    cam = tiny_camera(*size, bg=(0.2, 0.4, 0.6))
    say("case device pair count %dx%d" % size)
    cs = gs.camera_struct(cam)
    st = gs.SceneTensors(sc)
    g = torch.from_numpy(inputs.make_upstream_grad(cam.width, cam.height, 0)).cuda()
    host = gs.Frame(sc.n, cam.width, cam.height, gs.GS_APP_SH3, 1 << 14, want_tile_ids=True)
    P = host.forward(cs, st)
    dev = gs.Frame(sc.n, cam.width, cam.height, gs.GS_APP_SH3, 1 << 14, want_tile_ids=True)
    assert dev.forward(cs, st, sync_pairs=False) is None
    torch.cuda.synchronize()
    assert int(dev.num_pairs.item()) == P and not dev.pairs_overflowed()
    for k in ("values", "tile_ids"):
        assert torch.equal(getattr(dev, k)[:P], getattr(host, k)[:P]), k
    for k in ("ranges", "image", "final_T", "n_contrib"):
        assert torch.equal(getattr(dev, k), getattr(host, k)), k
    host.backward(cs, st, g)
    dev.backward(cs, st, g)
    torch.cuda.synchronize()
    for k in ("dmeans", "dlog_scales", "dquats", "dopacity_logits", "dsh"):
        a, b = getattr(dev, k).double(), getattr(host, k).double()
        assert torch.allclose(a, b, rtol=1e-5, atol=1e-12 + 1e-6 * float(b.abs().max())), k
    # overflow found on the device
    small = gs.Frame(sc.n, cam.width, cam.height, gs.GS_APP_SH3, P // 3)
    small.forward(cs, st, sync_pairs=False)
    torch.cuda.synchronize()
    assert small.pairs_overflowed() and int(small.num_pairs.item()) == P
    assert int(small.ranges.abs().sum().item()) == 0
    bg = torch.tensor([0.2, 0.4, 0.6], device="cuda").view(3, 1, 1).expand_as(small.image)
    assert torch.equal(small.image, bg.float())
    assert bool((small.final_T == 1).all()) and int(small.n_contrib.sum().item()) == 0
    small.backward(cs, st, g)
    torch.cuda.synchronize()
    for k in ("dmeans", "dlog_scales", "dquats", "dopacity_logits", "dsh"):
        assert int(torch.count_nonzero(getattr(small, k)[..., : sc.n]).item()) == 0, k
    # a host-mode count that understates P, with a capacity to match it: the
    # lists need more than the capacity, which is found on the device, and every
    # range comes out empty (nothing is written past the capacity)
    low = gs.Frame(sc.n, cam.width, cam.height, gs.GS_APP_SH3, P // 2)
    gs.gs_preprocess(cs, st.gaussians(), st.appearance(gs.GS_APP_SH3, 3), low.pre, low.workspace, low.ws_bytes,
                     sync_pairs=False)
    guard = torch.full((64,), -7, dtype=torch.int32, device="cuda")
    values = torch.cat([low.values, guard])
    gs.gs_bin_sort(cs, low.pre, sc.n, P // 2, P // 2, values, None, low.ranges, low.workspace, low.ws_bytes)
    torch.cuda.synchronize()
    assert int(low.ranges.abs().sum().item()) == 0
    assert torch.equal(values[P // 2:], guard)
    # retry with room for every pair
    retry = gs.Frame(sc.n, cam.width, cam.height, gs.GS_APP_SH3, P, want_tile_ids=True)
    retry.forward(cs, st, sync_pairs=False)
    torch.cuda.synchronize()
    assert not retry.pairs_overflowed()
    assert torch.equal(retry.values[:P], host.values[:P]) and torch.equal(retry.image, host.image)


# ---- the blend's work counts (measurement) ------------------------------------------

@pytest.mark.parametrize("case", ["tiny", "ragged", "medium"])
def test_render_work_counts(case):
    # gs_render_work: blended and visited entries against the oracle's
    # per-pixel counts (exactly where no pixel is flagged; otherwise within the
    # flagged pixels' list lengths), the listed entries equal to the sum of the
    # GPU's own n_contrib, and evaluated counts between them
    if case == "medium":
        sc, cam = inputs.make_scene("medium"), inputs.make_cameras("medium")[3]
    else:
        sc = inputs.make_scene("tiny")
        cam = inputs.make_cameras("tiny")[0] if case == "tiny" else tiny_camera(50, 37)
    say("case render work %s" % case)
    ref = orc.render(cam, sc, mode="f32")
    gpu = run_gpu(sc, cam)
    fr = gpu["frame"]
    counts = torch.zeros(5, dtype=torch.int64, device="cuda")
    gs.gs_render_work(gs.camera_struct(cam), fr.pre, sc.n, fr.values, fr.ranges, counts)
    torch.cuda.synchronize()
    blended, listed, ev_bwd, ev_fwd, walked = (int(v) for v in counts.cpu().numpy())
    say("  blended %d listed %d evaluated bwd %d fwd %d visited fwd %d" % (blended, listed, ev_bwd, ev_fwd, walked))
    assert listed == int(gpu["n_contrib"].astype(np.int64).sum())
    flagged = ref["margin"] <= 1.0
    ref_blended = int(ref["n_blended"].astype(np.int64).sum())
    ref_walked = int(ref["n_walked"].astype(np.int64).sum())
    tiles_x = (cam.width + 15) // 16
    ys, xs = np.mgrid[0:cam.height, 0:cam.width]
    lens = (ref["ranges"][:, 1] - ref["ranges"][:, 0])[(ys // 16) * tiles_x + xs // 16]
    slack = int(ref["n_contrib"][flagged].astype(np.int64).sum() + gpu["n_contrib"][flagged].astype(np.int64).sum())
    if not flagged.any():
        assert blended == ref_blended and walked == ref_walked
    assert abs(blended - ref_blended) <= slack
    assert abs(walked - ref_walked) <= int(lens[flagged].astype(np.int64).sum())
    assert blended <= ev_bwd <= listed and ev_bwd <= ev_fwd <= walked and listed <= walked


# ---- decoder weights far from their initialisation -----------------------------------

@pytest.mark.parametrize("kind,arch,factor", [("latent", None, 4.0), ("neural", (2, 16, 0), 4.0),
                                              ("neural", (3, 16, 0), 4.0), ("neural", (2, 32, 0), 4.0),
                                              ("neural", (3, 16, 0), 16.0)])
def test_decoder_large_weights(kind, arch, factor):
    # every decoder weight times 4 or 16 (exact in binary16): the backward's hidden-
    # layer gradients grow by the layers' norms on the way back and must stay
    # within binary16 range (the chunk's gradient scale accounts for them).
    # The binary16 rounding flips of the forward grow with the weights too, so
    # the colour and gradient bars are those of the decoder path scaled by the
    # weights' growth along the network (the factor per layer).
    sc = inputs.make_scene("tiny", appearance=(kind,), neural_arch=arch)
    attr = "mlp_w" if kind == "latent" else "neural_w"
    w = getattr(sc, attr).view(np.float16).astype(np.float32) * factor
    setattr(sc, attr, w.astype(np.float16).view(np.uint16))
    layers = 3 if kind == "latent" else arch[0] + 1
    growth = factor ** layers
    cam = tiny_camera()
    say("case large weights %s %s x%g" % (kind, arch, factor))
    ref = orc.render(cam, sc, kind=kind, sh_degree=3, mode="f32", half_act=True)
    flagged = flagged_pixels(ref["margin"])
    g = (inputs.make_upstream_grad(cam.width, cam.height, 0) * ~flagged[None]).astype(np.float32)
    grads = orc.render_bwd(cam, sc, ref["pre"], ref["ranges"], ref["values"], g, kind=kind, sh_degree=3, mode="f32",
                           half_act=True)
    gpu = run_gpu(sc, cam, kind, 3, g)
    vis = ref["pre"]["tiles"] > 0
    err = np.abs(gpu["splat"]["color"][:, vis] - ref["pre"]["color"][:, vis])
    say("  colours: max abs %.2e" % err.max())
    assert err.max() <= MLP_HALF_ATOL * growth
    for k, v in gpu["grads"].items():
        assert np.all(np.isfinite(v)), k
    st = grad_stats(gpu["grads"], grads)
    report_grads(st)
    for k, (rel, _, _, _) in st.items():
        assert rel <= 5e-3, (k, rel)
