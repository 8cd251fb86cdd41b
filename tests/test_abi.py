"""The C ABI without a GPU: the library loads, exports every entry point that
include/gsraster.h declares, sizes workspaces, and rejects bad arguments on the
host before launching anything."""
import ctypes as C
import os
import re
import subprocess

import pytest

from paper_2609_05255_amd import build as gsbuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gsraster.h")


@pytest.fixture(scope="module")
def gs():
    if not os.path.exists(gsbuild.LIB):
        gsbuild.build()
    from paper_2609_05255_amd import gsraster
    return gsraster


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gs_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_function(gs):
    names = declared_functions()
    assert {"gs_preprocess", "gs_bin_sort", "gs_render_fwd", "gs_render_bwd"} <= set(names)
    out = subprocess.run(["nm", "-D", "--defined-only", gs.LIB_PATH], capture_output=True, text=True, check=True)
    exported = set(re.findall(r"\bT (gs_[a-z0-9_]+)\b", out.stdout))
    assert set(names) <= exported, set(names) - exported
    lib = gs.lib()
    for name in names:
        assert getattr(lib, name) is not None


def test_version_and_kernel_names(gs):
    assert b"gfx950" in gs.lib().gs_version()
    assert [gs.lib().gs_kernel_name(i).decode() for i in range(len(gs.KERNEL_NAMES))] == gs.KERNEL_NAMES


def test_workspace_size(gs):
    a = gs.gs_workspace_size(1000, 64, 64, 10_000, gs.GS_APP_SH3)
    b = gs.gs_workspace_size(1000, 64, 64, 20_000, gs.GS_APP_SH3)
    c = gs.gs_workspace_size(1000, 64, 64, 10_000, gs.GS_APP_LATENT_MLP)
    assert 0 < a < b and a < c
    # four pair buffers of u32 per unit of capacity
    assert b - a >= 4 * 4 * 10_000
    with pytest.raises(gs.GsError) as e:
        gs.gs_workspace_size(-1, 64, 64, 10, gs.GS_APP_SH3)
    assert e.value.status == gs.GS_ERR_INVALID_ARG
    with pytest.raises(gs.GsError):
        gs.gs_workspace_size(10, 64, 64, 10, 7)
    with pytest.raises(gs.GsError):
        gs.gs_workspace_size(10, 64, 64, 1 << 32, gs.GS_APP_SH3)
    # the bin-sort's per-block buffers (4x4-tile blocks, and the segment table
    # bounded by capacity / 2048 + blocks) grow with the image
    big = gs.gs_workspace_size(1000, 4096, 4096, 10_000, gs.GS_APP_SH3)
    assert big - a >= 4 * 2 * (256 * 256 - 1)


def test_bin_sort_workspace_follows_the_image(gs):
    # a workspace sized for a small image is too small for a large one
    lib = gs.lib()
    pre = gs.Preprocessed(FAKE, FAKE, FAKE, FAKE)
    small = gs.gs_workspace_size(10, 64, 48, 100, gs.GS_APP_SH3)
    large = gs.gs_workspace_size(10, 4096, 4096, 100, gs.GS_APP_SH3)
    assert large > small
    cam = _camera(gs, width=4096, height=4096)
    st = lib.gs_bin_sort(C.byref(cam), C.byref(pre), 10, 10, 100, C.c_void_p(FAKE), None, C.c_void_p(FAKE),
                         C.c_void_p(FAKE * 256), small, None)
    assert st == gs.GS_ERR_CAPACITY and b"workspace" in lib.gs_last_error()


def test_bin_sort_rejects_more_than_65536_blocks(gs):
    # a block id shares a 32-bit key with the 16-bit mask of its tiles: at most
    # 65536 blocks of 4x4 tiles (1025 x 1025 tiles need 257 x 257 blocks)
    lib = gs.lib()
    pre = gs.Preprocessed(FAKE, FAKE, FAKE, FAKE)
    for side, want in ((16384, gs.GS_ERR_CAPACITY), (16400, gs.GS_ERR_UNSUPPORTED)):
        cam = _camera(gs, width=side, height=side)
        st = lib.gs_bin_sort(C.byref(cam), C.byref(pre), 10, 10, 100, C.c_void_p(FAKE), None, C.c_void_p(FAKE),
                             C.c_void_p(FAKE * 256), 1 << 20, None)
        assert st == want, (side, st, lib.gs_last_error())


def _camera(gs, **kw):
    from paper_2609_05255_amd import inputs
    c = gs.camera_struct(inputs.look_at_camera([0, 0, -3], 64, 48))
    for k, v in kw.items():
        setattr(c, k, v)
    return c


FAKE = 1 << 20   # a non-NULL pointer value; never dereferenced by argument checks


def test_preprocess_rejects_bad_arguments(gs):
    lib = gs.lib()
    g = gs.Gaussians(10, FAKE, FAKE, FAKE, FAKE)
    app = gs.Appearance(gs.GS_APP_SH3, 3, FAKE, None, None)
    pre = gs.Preprocessed(FAKE, FAKE, FAKE, FAKE)
    ok_cam = _camera(gs)

    def call(cam=ok_cam, g=g, app=app, pre=pre, ws=FAKE * 256, wsb=1 << 40):
        return lib.gs_preprocess(C.byref(cam) if cam is not None else None, C.byref(g) if g is not None else None,
                                 C.byref(app), C.byref(pre), None, C.c_void_p(ws), wsb, None)

    assert call(cam=None) == gs.GS_ERR_INVALID_ARG
    assert b"camera" in lib.gs_last_error()
    assert call(cam=_camera(gs, width=0)) == gs.GS_ERR_INVALID_ARG
    assert call(cam=_camera(gs, fx=0.0)) == gs.GS_ERR_INVALID_ARG
    assert call(cam=_camera(gs, width=1 << 20)) == gs.GS_ERR_INVALID_ARG
    assert call(g=gs.Gaussians(-1, FAKE, FAKE, FAKE, FAKE)) == gs.GS_ERR_INVALID_ARG
    assert call(g=gs.Gaussians(1 << 31, FAKE, FAKE, FAKE, FAKE)) == gs.GS_ERR_INVALID_ARG
    assert call(g=gs.Gaussians(10, None, FAKE, FAKE, FAKE)) == gs.GS_ERR_INVALID_ARG
    assert call(app=gs.Appearance(gs.GS_APP_SH3, 4, FAKE, None, None)) == gs.GS_ERR_INVALID_ARG
    assert b"sh_degree" in lib.gs_last_error()
    assert call(app=gs.Appearance(gs.GS_APP_SH3, 3, None, None, None)) == gs.GS_ERR_INVALID_ARG
    assert call(app=gs.Appearance(gs.GS_APP_LATENT_MLP, 0, None, FAKE, None)) == gs.GS_ERR_INVALID_ARG
    assert call(app=gs.Appearance(9, 0, FAKE, FAKE, FAKE)) == gs.GS_ERR_INVALID_ARG
    # neural: base colour always, features and weights once the residual is on, degree 0..3
    assert call(app=gs.Appearance(gs.GS_APP_NEURAL, 3, None, None, FAKE, None, FAKE)) == gs.GS_ERR_INVALID_ARG
    assert call(app=gs.Appearance(gs.GS_APP_NEURAL, 2, None, None, FAKE, FAKE, None)) == gs.GS_ERR_INVALID_ARG
    assert call(app=gs.Appearance(gs.GS_APP_NEURAL, 4, None, None, FAKE, FAKE, FAKE)) == gs.GS_ERR_INVALID_ARG
    # neural configurations: 1..3 hidden layers of 16, raw features; 32 wide only as the table's
    # 2-hidden-layer decoder on encoded features
    arch = lambda L, W, raw: gs.Appearance(gs.GS_APP_NEURAL, 3, None, None, FAKE, FAKE, FAKE, None, None, 0, L, W, raw)
    assert call(app=arch(4, 0, 0)) == gs.GS_ERR_INVALID_ARG
    assert call(app=arch(2, 8, 0)) == gs.GS_ERR_INVALID_ARG
    assert call(app=arch(3, 32, 0)) == gs.GS_ERR_UNSUPPORTED
    assert call(app=arch(2, 32, 1)) == gs.GS_ERR_UNSUPPORTED
    assert call(app=arch(2, 16, 2)) == gs.GS_ERR_INVALID_ARG
    folded_arch = gs.Appearance(gs.GS_APP_NEURAL_FOLDED, 3, None, None, FAKE, FAKE, None, FAKE, None, 0, 3, 0, 0)
    assert call(app=folded_arch) == gs.GS_ERR_INVALID_ARG
    folded_wide = gs.Appearance(gs.GS_APP_NEURAL_FOLDED, 3, None, None, FAKE, FAKE, None, FAKE, None, 0, 2, 32, 0)
    assert call(app=folded_wide) == gs.GS_ERR_INVALID_ARG
    # folded neural: pre-activations instead of features, 8-byte aligned
    folded = lambda deg, pre_act: gs.Appearance(gs.GS_APP_NEURAL_FOLDED, deg, None, None, FAKE, FAKE, None, pre_act)
    assert call(app=folded(3, None)) == gs.GS_ERR_INVALID_ARG
    assert b"preact" in lib.gs_last_error()
    assert call(app=folded(3, FAKE + 2)) == gs.GS_ERR_INVALID_ARG
    assert call(app=folded(4, FAKE)) == gs.GS_ERR_INVALID_ARG
    # lobes: base colour always, the lobe parameters once the lobe is on
    lobe = lambda kind, deg, base, lobes: gs.Appearance(kind, deg, None, None, None, base, None, None, lobes)
    for kind in (gs.GS_APP_NASG, gs.GS_APP_NASGABOR):
        assert call(app=lobe(kind, 1, FAKE, None)) == gs.GS_ERR_INVALID_ARG
        assert b"lobes" in lib.gs_last_error()
        assert call(app=lobe(kind, 0, None, FAKE)) == gs.GS_ERR_INVALID_ARG
        assert call(app=lobe(kind, 4, FAKE, FAKE)) == gs.GS_ERR_INVALID_ARG
    assert call(pre=gs.Preprocessed(FAKE, FAKE, FAKE, None)) == gs.GS_ERR_INVALID_ARG
    assert call(ws=FAKE + 4) == gs.GS_ERR_INVALID_ARG              # misaligned workspace
    assert call(wsb=16) == gs.GS_ERR_CAPACITY
    assert b"workspace" in lib.gs_last_error()


def test_bin_sort_reports_capacity(gs):
    lib = gs.lib()
    cam = _camera(gs)
    pre = gs.Preprocessed(FAKE, FAKE, FAKE, FAKE)
    st = lib.gs_bin_sort(C.byref(cam), C.byref(pre), 10, 5000, 4000, C.c_void_p(FAKE), None, C.c_void_p(FAKE),
                         C.c_void_p(FAKE * 256), 1 << 40, None)
    assert st == gs.GS_ERR_CAPACITY
    assert b"5000" in lib.gs_last_error() and b"4000" in lib.gs_last_error()
    st = lib.gs_bin_sort(C.byref(cam), C.byref(pre), 10, 10, 1 << 32, C.c_void_p(FAKE), None, C.c_void_p(FAKE),
                         C.c_void_p(FAKE * 256), 1 << 40, None)
    assert st == gs.GS_ERR_INVALID_ARG
    st = lib.gs_bin_sort(C.byref(cam), C.byref(pre), 10, 10, 100, C.c_void_p(FAKE), None, None,
                         C.c_void_p(FAKE * 256), 1 << 40, None)
    assert st == gs.GS_ERR_INVALID_ARG


def test_bin_sort_device_count_arguments(gs):
    # device mode (the pair count read on the device): nothing about P can be
    # checked on the host, but the buffers the capacity promises must exist
    lib = gs.lib()
    cam = _camera(gs)
    pre = gs.Preprocessed(FAKE, FAKE, FAKE, FAKE)
    st = lib.gs_bin_sort(C.byref(cam), C.byref(pre), 10, gs.GS_PAIRS_ON_DEVICE, 100, None, None, C.c_void_p(FAKE),
                         C.c_void_p(FAKE * 256), 1 << 40, None)
    assert st == gs.GS_ERR_INVALID_ARG and b"values" in lib.gs_last_error()
    st = lib.gs_bin_sort(C.byref(cam), C.byref(pre), 10, gs.GS_PAIRS_ON_DEVICE, 1 << 32, C.c_void_p(FAKE), None,
                         C.c_void_p(FAKE), C.c_void_p(FAKE * 256), 1 << 40, None)
    assert st == gs.GS_ERR_INVALID_ARG
    # the count lives in pre->num_pairs: required in either mode
    nopairs = gs.Preprocessed(FAKE, FAKE, FAKE, None)
    st = lib.gs_bin_sort(C.byref(cam), C.byref(nopairs), 10, gs.GS_PAIRS_ON_DEVICE, 100, C.c_void_p(FAKE), None,
                         C.c_void_p(FAKE), C.c_void_p(FAKE * 256), 1 << 40, None)
    assert st == gs.GS_ERR_INVALID_ARG


def test_timer_is_caller_owned(gs):
    # a timing context is created, attached, read, reset and destroyed by the
    # caller; without one attached the library records nothing
    lib = gs.lib()
    ms = (C.c_double * 4)()
    cnt = (C.c_int64 * 4)()
    assert lib.gs_timer_read(None, ms, cnt, 4) == gs.GS_ERR_INVALID_ARG
    assert lib.gs_timer_reset(None) == gs.GS_ERR_INVALID_ARG
    assert lib.gs_timer_attach(None) == gs.GS_OK
    assert lib.gs_timer_destroy(None) == gs.GS_OK
    assert lib.gs_timer_create(None) == gs.GS_ERR_INVALID_ARG


def test_render_calls_reject_bad_arguments(gs):
    lib = gs.lib()
    cam = _camera(gs)
    pre = gs.Preprocessed(FAKE, FAKE, FAKE, FAKE)
    st = lib.gs_render_fwd(C.byref(cam), C.byref(pre), 10, C.c_void_p(FAKE), C.c_void_p(FAKE), None,
                           C.c_void_p(FAKE), C.c_void_p(FAKE), None)
    assert st == gs.GS_ERR_INVALID_ARG
    g = gs.Gaussians(10, FAKE, FAKE, FAKE, FAKE)
    app = gs.Appearance(gs.GS_APP_SH3, 3, FAKE, None, None)
    grads = gs.Grads(FAKE, FAKE, FAKE, FAKE, None, None, None, None)
    st = lib.gs_render_bwd(C.byref(cam), C.byref(g), C.byref(app), C.byref(pre), C.c_void_p(FAKE), C.c_void_p(FAKE),
                           C.c_void_p(FAKE), C.c_void_p(FAKE), C.c_void_p(FAKE), C.byref(grads),
                           C.c_void_p(FAKE * 256), 1 << 40, None)
    assert st == gs.GS_ERR_INVALID_ARG and b"dsh" in lib.gs_last_error()
    # the folded neural form renders only
    app = gs.Appearance(gs.GS_APP_NEURAL_FOLDED, 3, None, None, FAKE, FAKE, None, FAKE)
    grads = gs.Grads(FAKE, FAKE, FAKE, FAKE, None, None, FAKE, None, FAKE, FAKE)
    st = lib.gs_render_bwd(C.byref(cam), C.byref(g), C.byref(app), C.byref(pre), C.c_void_p(FAKE), C.c_void_p(FAKE),
                           C.c_void_p(FAKE), C.c_void_p(FAKE), C.c_void_p(FAKE), C.byref(grads),
                           C.c_void_p(FAKE * 256), 1 << 40, None)
    assert st == gs.GS_ERR_INVALID_ARG and b"folded" in lib.gs_last_error()
    # lobes need both of their gradient arrays
    app = gs.Appearance(gs.GS_APP_NASG, 1, None, None, None, FAKE, None, None, FAKE)
    grads = gs.Grads(FAKE, FAKE, FAKE, FAKE, None, None, None, None, FAKE, None, None)
    st = lib.gs_render_bwd(C.byref(cam), C.byref(g), C.byref(app), C.byref(pre), C.c_void_p(FAKE), C.c_void_p(FAKE),
                           C.c_void_p(FAKE), C.c_void_p(FAKE), C.c_void_p(FAKE), C.byref(grads),
                           C.c_void_p(FAKE * 256), 1 << 40, None)
    assert st == gs.GS_ERR_INVALID_ARG and b"dlobes" in lib.gs_last_error()


def test_render_bwd_adam_rejects_bad_arguments(gs):
    lib = gs.lib()
    cam = _camera(gs)
    pre = gs.Preprocessed(FAKE, FAKE, FAKE, FAKE)
    g = gs.Gaussians(10, FAKE, 2 * FAKE, 3 * FAKE, 4 * FAKE)
    sh = 5 * FAKE
    app = gs.Appearance(gs.GS_APP_SH3, 3, sh, None, None)
    grads = gs.Grads()
    lr = (C.c_float * 48)(*([1e-3] * 48))

    def tensors(params=(FAKE, 2 * FAKE, 3 * FAKE, 4 * FAKE, sh), rows=(3, 3, 4, 1, 48), n=10, m=6 * FAKE):
        arr = (gs.AdamTensor * gs.GS_RENDER_ADAM_TENSORS)()
        for k in range(gs.GS_RENDER_ADAM_TENSORS):
            arr[k] = gs.AdamTensor(params[k], None, m, 7 * FAKE, None, n, rows[k], 0.999,
                                   C.cast(lr, C.POINTER(C.c_float)))
        return arr

    def call(app=app, adam=tensors(), beta1=0.9, eps=1e-15, step=1):
        return lib.gs_render_bwd_adam(C.byref(cam), C.byref(g), C.byref(app), C.byref(pre), C.c_void_p(FAKE),
                                      C.c_void_p(FAKE), C.c_void_p(FAKE), C.c_void_p(FAKE), C.c_void_p(FAKE),
                                      C.byref(grads), adam, beta1, eps, step, C.c_void_p(FAKE * 256), 1 << 40, None)

    # the step inside the backward is built for SH3 only
    latent = gs.Appearance(gs.GS_APP_LATENT_MLP, 3, None, FAKE, FAKE)
    assert call(app=latent) == gs.GS_ERR_UNSUPPORTED
    assert call(adam=None) == gs.GS_ERR_INVALID_ARG
    assert call(step=0) == gs.GS_ERR_INVALID_ARG
    assert call(beta1=1.0) == gs.GS_ERR_INVALID_ARG
    assert call(eps=0.0) == gs.GS_ERR_INVALID_ARG
    # each tensor must be the parameter array it updates, with its rows and n
    assert call(adam=tensors(params=(FAKE, 2 * FAKE, 3 * FAKE, 4 * FAKE, 9 * FAKE))) == gs.GS_ERR_INVALID_ARG
    assert b"param" in lib.gs_last_error()
    assert call(adam=tensors(rows=(3, 3, 4, 1, 47))) == gs.GS_ERR_INVALID_ARG
    assert call(adam=tensors(n=11)) == gs.GS_ERR_INVALID_ARG
    assert call(adam=tensors(m=None)) == gs.GS_ERR_INVALID_ARG and b"moment" in lib.gs_last_error()


def test_neural_fold_rejects_bad_arguments(gs):
    lib = gs.lib()
    f = lambda *a: lib.gs_neural_fold(*[C.c_void_p(x) if x is not None else None for x in a[:2]], a[2],
                                      C.c_void_p(a[3]) if a[3] is not None else None, None)
    assert f(FAKE, FAKE, -1, FAKE) == gs.GS_ERR_INVALID_ARG
    assert f(FAKE, FAKE, 1 << 31, FAKE) == gs.GS_ERR_INVALID_ARG
    assert f(None, FAKE, 10, FAKE) == gs.GS_ERR_INVALID_ARG
    assert f(FAKE, FAKE, 10, None) == gs.GS_ERR_INVALID_ARG
    assert f(FAKE, FAKE, 10, FAKE + 4) == gs.GS_ERR_INVALID_ARG
    assert b"aligned" in lib.gs_last_error()
    assert f(None, None, 0, None) == gs.GS_OK          # nothing to do, nothing launched
    # the folded form has no backward, so its workspace holds no weight-gradient partials
    assert gs.gs_workspace_size(1000, 64, 64, 100, gs.GS_APP_NEURAL_FOLDED) < \
        gs.gs_workspace_size(1000, 64, 64, 100, gs.GS_APP_NEURAL)


def test_adam_rejects_bad_arguments(gs):
    # every case fails a host check, so the fake pointers are never used
    t = dict(param=FAKE, grad=FAKE, exp_avg=FAKE, exp_avg_sq=FAKE, rows=2, n=10, beta2=0.999, lr=[1e-3, 1e-3])
    cases = [(dict(rows=0, lr=[]), {}), (dict(beta2=1.0), {}), (dict(lr=None), {}), (dict(n=-1), {}),
             (dict(grad=None), {}), ({}, dict(step=0)), ({}, dict(beta1=1.0)), ({}, dict(eps=0.0))]
    for bad, kw in cases:
        args = dict(beta1=0.9, eps=1e-8, step=1, stream=0)
        args.update(kw)
        with pytest.raises(gs.GsError) as e:
            gs.gs_adam_step([dict(t, **bad)], **args)
        assert e.value.status == gs.GS_ERR_INVALID_ARG, (bad, kw)
    with pytest.raises(gs.GsError):
        gs.gs_adam_step([], 0.9, 1e-8, 1, stream=0)
    with pytest.raises(gs.GsError):     # 129 rows in total
        gs.gs_adam_step([dict(t, rows=65, lr=[1e-3] * 65), dict(t, rows=64, lr=[1e-3] * 64)], 0.9, 1e-8, 1,
                        stream=0)
    with pytest.raises(gs.GsError):     # nine tensors
        gs.gs_adam_step([t] * 9, 0.9, 1e-8, 1, stream=0)


def test_preprocess_noalloc_limit(gs):
    # sizes beyond the static scratch are refused on the host, before any device work
    lib = gs.lib()
    cam = _camera(gs)
    pre = gs.Preprocessed(FAKE, FAKE, FAKE, FAKE)
    app = gs.Appearance(gs.GS_APP_SH3, 3, FAKE, None, None)
    g = gs.Gaussians((1 << 24) + 1, FAKE, FAKE, FAKE, FAKE)
    assert lib.gs_preprocess_noalloc(C.byref(cam), C.byref(g), C.byref(app), C.byref(pre), None, None) == \
        gs.GS_ERR_CAPACITY
    assert b"at most 16777216" in lib.gs_last_error()
    g = gs.Gaussians(10, FAKE, None, FAKE, FAKE)
    assert lib.gs_preprocess_noalloc(C.byref(cam), C.byref(g), C.byref(app), C.byref(pre), None, None) == \
        gs.GS_ERR_INVALID_ARG
