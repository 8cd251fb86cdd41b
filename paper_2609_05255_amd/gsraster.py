"""Python binding of libgsraster.so (the C ABI of include/gsraster.h).

Argument marshalling only: torch tensors provide device memory and the stream,
every step of the rasterizer runs in the HIP library. The library must have
been built (``python -m paper_2609_05255_amd.build``); importing this module
raises if it is missing, there is no fallback.

Function names follow the C ABI: gs_preprocess, gs_bin_sort, gs_render_fwd,
gs_render_bwd, gs_workspace_size. ``Frame`` owns the buffers of one camera's
forward + backward pass for a scene of n Gaussians.
"""
from __future__ import annotations

import ctypes as C
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgsraster.so")

GS_OK, GS_ERR_INVALID_ARG, GS_ERR_CAPACITY, GS_ERR_DEVICE, GS_ERR_UNSUPPORTED = range(5)
GS_PAIRS_ON_DEVICE = (1 << 64) - 1   # gs_bin_sort reads the pair count on the device
GS_APP_SH3, GS_APP_LATENT_MLP, GS_APP_NEURAL, GS_APP_NEURAL_FOLDED, GS_APP_NASG, GS_APP_NASGABOR = range(6)
LOBE_ROWS = {GS_APP_NASG: 8, GS_APP_NASGABOR: 9}
NEURAL_FEATURES = 8
NEURAL_WEIGHTS = 816


def neural_weight_count(arch=None) -> int:
    """Weights of the neural decoder with arch = (hidden layers, width, raw16); None: the paper's (2, 16, 0)."""
    layers, width = (2, 16) if arch is None else (int(arch[0]), int(arch[1]))
    return 32 * width + (layers - 1) * width * width + 3 * width
KERNEL_NAMES = ["preprocess", "pair_count", "depth_sort", "entry_offsets", "block_entries", "block_sort", "tile_lists",
                "blend_fwd", "bwd_prep", "blend_bwd", "preprocess_bwd", "mlp_reduce", "adam", "neural_fold"]
ADAM_MAX_TENSORS = 8
ADAM_MAX_ROWS = 128
SPLAT_BYTES = 64
MLP_WEIGHTS = 1664


class GsError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("gsraster status %d: %s" % (status, msg))
        self.status = status


# gs_splat's fields as 4-byte word offsets into its 64-byte record (the four
# int16 of the rectangle fill words 12 and 13)
SPLAT_WORDS = dict(mean_x=0, mean_y=1, conic_a=2, conic_b=3, conic_c=4, opacity=5, color=6, power_min=9,
                   ext_x=10, ext_y=11, rect=12, depth=14)


class Camera(C.Structure):
    _fields_ = [("viewmat", C.c_float * 12), ("campos", C.c_float * 3), ("fx", C.c_float), ("fy", C.c_float),
                ("cx", C.c_float), ("cy", C.c_float), ("width", C.c_int32), ("height", C.c_int32),
                ("near_plane", C.c_float), ("bg", C.c_float * 3)]


class Gaussians(C.Structure):
    _fields_ = [("n", C.c_int64), ("means", C.c_void_p), ("log_scales", C.c_void_p), ("quats", C.c_void_p),
                ("opacity_logits", C.c_void_p)]


class Appearance(C.Structure):
    _fields_ = [("kind", C.c_int32), ("sh_degree", C.c_int32), ("sh", C.c_void_p), ("latent", C.c_void_p),
                ("mlp_w", C.c_void_p), ("base_color", C.c_void_p), ("features", C.c_void_p),
                ("preact", C.c_void_p), ("lobes", C.c_void_p), ("sh_y0_folded", C.c_int32),
                ("neural_layers", C.c_int32), ("neural_width", C.c_int32), ("neural_raw16", C.c_int32)]


class Preprocessed(C.Structure):
    _fields_ = [("splats", C.c_void_p), ("tiles_touched", C.c_void_p), ("depth_key", C.c_void_p),
                ("num_pairs", C.c_void_p), ("color_jac", C.c_void_p)]


class Grads(C.Structure):
    _fields_ = [("dmeans", C.c_void_p), ("dlog_scales", C.c_void_p), ("dquats", C.c_void_p),
                ("dopacity_logits", C.c_void_p), ("dsh", C.c_void_p), ("dlatent", C.c_void_p),
                ("dmlp_w", C.c_void_p), ("dmean2d", C.c_void_p), ("dbase_color", C.c_void_p),
                ("dfeatures", C.c_void_p), ("dlobes", C.c_void_p)]


class AdamTensor(C.Structure):
    _fields_ = [("param", C.c_void_p), ("grad", C.c_void_p), ("exp_avg", C.c_void_p), ("exp_avg_sq", C.c_void_p),
                ("param_half", C.c_void_p), ("n", C.c_int64), ("rows", C.c_int32), ("beta2", C.c_float),
                ("lr", C.POINTER(C.c_float))]


_lib = None


def lib() -> C.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libgsraster.so is not built (python -m paper_2609_05255_amd.build)")
        L = C.CDLL(LIB_PATH)
        vp, i32, i64, u64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_uint64, C.c_size_t
        P = C.POINTER
        L.gs_preprocess.argtypes = [P(Camera), P(Gaussians), P(Appearance), P(Preprocessed), P(u64), vp, sz, vp]
        L.gs_preprocess_noalloc.argtypes = [P(Camera), P(Gaussians), P(Appearance), P(Preprocessed), P(u64), vp]
        L.gs_bin_sort.argtypes = [P(Camera), P(Preprocessed), i64, u64, u64, vp, vp, vp, vp, sz, vp]
        L.gs_render_fwd.argtypes = [P(Camera), P(Preprocessed), i64, vp, vp, vp, vp, vp, vp]
        L.gs_render_work.argtypes = [P(Camera), P(Preprocessed), i64, vp, vp, vp, vp]
        L.gs_render_bwd.argtypes = [P(Camera), P(Gaussians), P(Appearance), P(Preprocessed), vp, vp, vp, vp, vp,
                                    P(Grads), vp, sz, vp]
        L.gs_workspace_size.argtypes = [i64, i32, i32, u64, i32, P(sz)]
        L.gs_mlp_eval.argtypes = [vp, i64, vp, vp, vp]
        L.gs_neural_fold.argtypes = [vp, vp, i64, vp, vp]
        L.gs_adam_step.argtypes = [P(AdamTensor), i32, C.c_float, C.c_float, i64, vp]
        L.gs_render_bwd_adam.argtypes = [P(Camera), P(Gaussians), P(Appearance), P(Preprocessed), vp, vp, vp, vp,
                                         vp, P(Grads), P(AdamTensor), C.c_float, C.c_float, i64, vp, sz, vp]
        L.gs_timer_create.argtypes = [P(vp)]
        L.gs_timer_destroy.argtypes = [vp]
        L.gs_timer_attach.argtypes = [vp]
        L.gs_timer_reset.argtypes = [vp]
        L.gs_timer_read.argtypes = [vp, P(C.c_double), P(i64), i32]
        for f in ("gs_preprocess", "gs_preprocess_noalloc", "gs_bin_sort", "gs_render_fwd", "gs_render_work",
                  "gs_render_bwd", "gs_render_bwd_adam", "gs_workspace_size", "gs_mlp_eval", "gs_neural_fold",
                  "gs_adam_step", "gs_timer_create", "gs_timer_destroy", "gs_timer_attach", "gs_timer_reset",
                  "gs_timer_read"):
            getattr(L, f).restype = C.c_int
        L.gs_last_error.restype = C.c_char_p
        L.gs_version.restype = C.c_char_p
        L.gs_kernel_name.restype = C.c_char_p
        L.gs_kernel_name.argtypes = [i32]
        _lib = L
    return _lib


def _check(status: int):
    if status != GS_OK:
        raise GsError(status, lib().gs_last_error().decode())


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return C.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        return C.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return C.c_void_p(stream.cuda_stream)
    return C.c_void_p(stream)


def camera_struct(cam) -> Camera:
    c = Camera()
    vm = [float(v) for v in list(cam.viewmat.reshape(-1))]
    for k in range(12):
        c.viewmat[k] = vm[k]
    for k in range(3):
        c.campos[k] = float(cam.campos[k])
        c.bg[k] = float(cam.bg[k])
    c.fx, c.fy, c.cx, c.cy = float(cam.fx), float(cam.fy), float(cam.cx), float(cam.cy)
    c.width, c.height = int(cam.width), int(cam.height)
    c.near_plane = float(cam.near)
    return c


class SceneTensors:
    """Scene parameters resident on the GPU (planar, contiguous)."""

    def __init__(self, scene, device="cuda"):
        f32 = lambda a: torch.from_numpy(a).to(device=device, dtype=torch.float32).contiguous()
        h16 = lambda a: torch.from_numpy(a.view("int16")).to(device=device).contiguous()
        self.n = int(scene.n)
        self.means = f32(scene.means)
        self.log_scales = f32(scene.log_scales)
        self.quats = f32(scene.quats)
        self.opacity_logits = f32(scene.opacity_logits)
        self.sh = f32(scene.sh) if getattr(scene, "sh", None) is not None else None
        self.latent = h16(scene.latent) if getattr(scene, "latent", None) is not None else None
        self.mlp_w = h16(scene.mlp_w) if getattr(scene, "mlp_w", None) is not None else None
        self.base_color = f32(scene.base_color) if getattr(scene, "base_color", None) is not None else None
        self.features = h16(scene.features) if getattr(scene, "features", None) is not None else None
        self.neural_w = h16(scene.neural_w) if getattr(scene, "neural_w", None) is not None else None
        self.preact = None   # [n][16] binary16 pre-activations of the folded form (fold_neural)
        self.sh_y0_folded = bool(getattr(scene, "sh_y0_folded", False))
        self.neural_arch = getattr(scene, "neural_arch", None)
        self.lobes = f32(scene.lobes) if getattr(scene, "lobes", None) is not None else None
        self.lobes_gabor = f32(scene.lobes_gabor) if getattr(scene, "lobes_gabor", None) is not None else None

    def fold_neural(self, stream=None):
        """Computes the folded form's per-Gaussian pre-activations (gs_neural_fold)."""
        if self.preact is None:
            self.preact = torch.empty((self.n, 16), dtype=torch.int16, device=self.features.device)
        gs_neural_fold(self.features, self.neural_w, self.n, self.preact, stream)
        return self.preact

    def gaussians(self) -> Gaussians:
        return Gaussians(self.n, _ptr(self.means), _ptr(self.log_scales), _ptr(self.quats),
                         _ptr(self.opacity_logits))

    def appearance(self, kind: int, sh_degree: int = 3) -> Appearance:
        if kind == GS_APP_NEURAL:
            layers, width, raw16 = self.neural_arch if self.neural_arch is not None else (0, 0, 0)
            return Appearance(kind, sh_degree, None, None, _ptr(self.neural_w), _ptr(self.base_color),
                              _ptr(self.features), None, None, 0, layers, width, raw16)
        if kind == GS_APP_NEURAL_FOLDED:
            if self.preact is None:
                raise RuntimeError("fold_neural() first: the folded form reads its pre-activations")
            return Appearance(kind, sh_degree, None, None, _ptr(self.neural_w), _ptr(self.base_color), None,
                              _ptr(self.preact), None)
        if kind in LOBE_ROWS:
            lobes = self.lobes_gabor if kind == GS_APP_NASGABOR else self.lobes
            return Appearance(kind, sh_degree, None, None, None, _ptr(self.base_color), None, None, _ptr(lobes))
        return Appearance(kind, sh_degree, _ptr(self.sh), _ptr(self.latent), _ptr(self.mlp_w), None, None, None,
                          None, int(self.sh_y0_folded))


def gs_workspace_size(n: int, width: int, height: int, capacity: int, kind: int) -> int:
    out = C.c_size_t(0)
    _check(lib().gs_workspace_size(n, width, height, capacity, kind, C.byref(out)))
    return out.value


def gs_preprocess(cam: Camera, g: Gaussians, app: Appearance, pre: Preprocessed, workspace, ws_bytes: int,
                  stream=None, sync_pairs: bool = True):
    p = C.c_uint64(0)
    _check(lib().gs_preprocess(C.byref(cam), C.byref(g), C.byref(app), C.byref(pre),
                               C.byref(p) if sync_pairs else None, _ptr(workspace), ws_bytes, _stream(stream)))
    return p.value if sync_pairs else None


def gs_preprocess_noalloc(cam: Camera, g: Gaussians, app: Appearance, pre: Preprocessed, stream=None,
                          sync_pairs: bool = True):
    """gs_preprocess without a workspace (the library's static per-GPU scratch)."""
    p = C.c_uint64(0)
    _check(lib().gs_preprocess_noalloc(C.byref(cam), C.byref(g), C.byref(app), C.byref(pre),
                                       C.byref(p) if sync_pairs else None, _stream(stream)))
    return p.value if sync_pairs else None


def gs_bin_sort(cam: Camera, pre: Preprocessed, n: int, num_pairs: int, capacity: int, values, tile_ids,
                tile_ranges, workspace, ws_bytes: int, stream=None):
    _check(lib().gs_bin_sort(C.byref(cam), C.byref(pre), n, num_pairs, capacity, _ptr(values), _ptr(tile_ids),
                             _ptr(tile_ranges), _ptr(workspace), ws_bytes, _stream(stream)))


def gs_render_fwd(cam: Camera, pre: Preprocessed, n: int, values, tile_ranges, image, final_T, n_contrib,
                  stream=None):
    _check(lib().gs_render_fwd(C.byref(cam), C.byref(pre), n, _ptr(values), _ptr(tile_ranges), _ptr(image),
                               _ptr(final_T), _ptr(n_contrib), _stream(stream)))


def gs_render_work(cam: Camera, pre: Preprocessed, n: int, values, tile_ranges, counts, stream=None):
    """counts: int64 device tensor [5] (blended, listed, evaluated backward, evaluated forward,
    visited forward)."""
    _check(lib().gs_render_work(C.byref(cam), C.byref(pre), n, _ptr(values), _ptr(tile_ranges), _ptr(counts),
                                _stream(stream)))


def gs_render_bwd(cam: Camera, g: Gaussians, app: Appearance, pre: Preprocessed, values, tile_ranges, final_T,
                  n_contrib, dL_dimage, grads: Grads, workspace, ws_bytes: int, stream=None):
    _check(lib().gs_render_bwd(C.byref(cam), C.byref(g), C.byref(app), C.byref(pre), _ptr(values),
                               _ptr(tile_ranges), _ptr(final_T), _ptr(n_contrib), _ptr(dL_dimage), C.byref(grads),
                               _ptr(workspace), ws_bytes, _stream(stream)))


def gs_mlp_eval(x, rows: int, mlp_w, colors, stream=None):
    _check(lib().gs_mlp_eval(_ptr(x), rows, _ptr(mlp_w), _ptr(colors), _stream(stream)))


def gs_neural_fold(features, neural_w, n: int, preact, stream=None):
    _check(lib().gs_neural_fold(_ptr(features), _ptr(neural_w), n, _ptr(preact), _stream(stream)))


def _adam_tensors(tensors):
    arr = (AdamTensor * max(1, len(tensors)))()
    keep = []
    for k, t in enumerate(tensors):
        lr = None
        if t["lr"] is not None:
            if len(t["lr"]) < int(t["rows"]):
                raise ValueError("lr needs one entry per row")
            lr = (C.c_float * len(t["lr"]))(*[float(x) for x in t["lr"]])
            keep.append(lr)
        arr[k] = AdamTensor(_ptr(t["param"]), _ptr(t.get("grad")), _ptr(t["exp_avg"]), _ptr(t["exp_avg_sq"]),
                            _ptr(t.get("param_half")), int(t["n"]), int(t["rows"]), float(t["beta2"]),
                            C.cast(lr, C.POINTER(C.c_float)) if lr is not None else None)
    return arr, keep


def gs_adam_step(tensors, beta1: float, eps: float, step: int, stream=None):
    """tensors: list of dicts with param, grad, exp_avg, exp_avg_sq (device fp32 [rows][n]), optional
    param_half (device int16/uint16 [rows][n]), rows, n, beta2 and lr (a sequence of `rows` floats)."""
    arr, keep = _adam_tensors(tensors)
    _check(lib().gs_adam_step(arr, len(tensors), float(beta1), float(eps), int(step), _stream(stream)))


GS_RENDER_ADAM_TENSORS = 5


def gs_render_bwd_adam(cam: Camera, g: Gaussians, app: Appearance, pre: Preprocessed, values, tile_ranges, final_T,
                       n_contrib, dL_dimage, grads: Grads, tensors, beta1: float, eps: float, step: int, workspace,
                       ws_bytes: int, stream=None):
    """tensors: the GS_RENDER_ADAM_TENSORS per-Gaussian tensors (dicts as for gs_adam_step, grad unused) in
    the order means, log_scales, quats, opacity_logits, sh."""
    if len(tensors) != GS_RENDER_ADAM_TENSORS:
        raise ValueError("gs_render_bwd_adam takes %d tensors" % GS_RENDER_ADAM_TENSORS)
    arr, keep = _adam_tensors(tensors)
    _check(lib().gs_render_bwd_adam(C.byref(cam), C.byref(g), C.byref(app), C.byref(pre), _ptr(values),
                                    _ptr(tile_ranges), _ptr(final_T), _ptr(n_contrib), _ptr(dL_dimage),
                                    C.byref(grads), arr, float(beta1), float(eps), int(step), _ptr(workspace),
                                    ws_bytes, _stream(stream)))


class Timer:
    """A caller-owned kernel-timing context (gs_timer_*): while attached to the
    calling thread, every kernel the library launches from it is timed."""

    def __init__(self):
        h = C.c_void_p()
        _check(lib().gs_timer_create(C.byref(h)))
        self.handle = h

    def attach(self):
        _check(lib().gs_timer_attach(self.handle))

    @staticmethod
    def detach():
        _check(lib().gs_timer_attach(None))

    def reset(self):
        _check(lib().gs_timer_reset(self.handle))

    def read(self) -> dict:
        k = len(KERNEL_NAMES)
        ms = (C.c_double * k)()
        cnt = (C.c_int64 * k)()
        _check(lib().gs_timer_read(self.handle, ms, cnt, k))
        return {KERNEL_NAMES[i]: (ms[i], cnt[i]) for i in range(k)}

    def close(self):
        if self.handle:
            _check(lib().gs_timer_destroy(self.handle))
            self.handle = None


_timer = None


def timing_enable(on: bool = True):
    """Attaches (on) or detaches (off) this module's timer to the calling thread."""
    global _timer
    if on:
        if _timer is None:
            _timer = Timer()
        _timer.attach()
    else:
        Timer.detach()


def timing_reset():
    _timer.reset()


def timing_read() -> dict:
    return _timer.read()


class Frame:
    """Device buffers for rendering one image of a scene and its backward pass."""

    def __init__(self, n: int, width: int, height: int, kind: int, capacity: int, device="cuda",
                 want_tile_ids: bool = False, want_dmean2d: bool = False, neural_arch=None):
        self.n, self.width, self.height, self.kind, self.capacity = n, width, height, kind, capacity
        d = device
        nn = max(n, 1)
        self.tiles_x, self.tiles_y = (width + 15) // 16, (height + 15) // 16
        self.splats = torch.empty(nn * SPLAT_BYTES // 4, dtype=torch.float32, device=d)
        self.tiles_touched = torch.empty(nn, dtype=torch.int32, device=d)
        self.depth_key = torch.empty(nn, dtype=torch.int32, device=d)
        self.num_pairs = torch.zeros(1, dtype=torch.int64, device=d)
        self.values = torch.empty(max(capacity, 1), dtype=torch.int32, device=d)
        self.tile_ids = torch.empty(max(capacity, 1), dtype=torch.int32, device=d) if want_tile_ids else None
        self.ranges = torch.empty(self.tiles_x * self.tiles_y * 2, dtype=torch.int32, device=d)
        self.image = torch.empty(3, height, width, dtype=torch.float32, device=d)
        self.final_T = torch.empty(height, width, dtype=torch.float32, device=d)
        self.n_contrib = torch.empty(height, width, dtype=torch.int32, device=d)
        self.ws_bytes = gs_workspace_size(n, width, height, capacity, kind)
        self.workspace = torch.empty(max(self.ws_bytes, 256) // 4 + 64, dtype=torch.float32, device=d)
        self.dmeans = torch.empty(3, nn, device=d)
        self.dlog_scales = torch.empty(3, nn, device=d)
        self.dquats = torch.empty(4, nn, device=d)
        self.dopacity_logits = torch.empty(nn, device=d)
        self.dsh = torch.empty(48, nn, device=d) if kind == GS_APP_SH3 else None
        self.dlatent = torch.empty(14, nn, device=d) if kind == GS_APP_LATENT_MLP else None
        self.dmlp_w = (torch.empty(MLP_WEIGHTS, device=d) if kind == GS_APP_LATENT_MLP else
                       torch.empty(neural_weight_count(neural_arch), device=d) if kind == GS_APP_NEURAL else None)
        self.dmean2d = torch.empty(2, nn, device=d) if want_dmean2d else None
        self.dbase_color = torch.empty(3, nn, device=d) if kind in (GS_APP_NEURAL, *LOBE_ROWS) else None
        raw16 = neural_arch is not None and bool(neural_arch[2])
        self.dfeatures = torch.empty(16 if raw16 else NEURAL_FEATURES, nn, device=d) if kind == GS_APP_NEURAL else None
        self.dlobes = torch.empty(LOBE_ROWS[kind], nn, device=d) if kind in LOBE_ROWS else None
        # SH3: the colour's view-direction Jacobian, for the backward (gs_preprocessed.color_jac)
        self.color_jac = torch.empty(10 * nn, dtype=torch.float32, device=d) if kind == GS_APP_SH3 else None
        self.pre = Preprocessed(_ptr(self.splats), _ptr(self.tiles_touched), _ptr(self.depth_key),
                                _ptr(self.num_pairs), _ptr(self.color_jac))
        self.grads = Grads(_ptr(self.dmeans), _ptr(self.dlog_scales), _ptr(self.dquats),
                           _ptr(self.dopacity_logits), _ptr(self.dsh), _ptr(self.dlatent), _ptr(self.dmlp_w),
                           _ptr(self.dmean2d), _ptr(self.dbase_color), _ptr(self.dfeatures), _ptr(self.dlobes))
        self.last_pairs = 0

    def forward(self, cam: Camera, scene: SceneTensors, sh_degree: int = 3, stream=None,
                sync_pairs: bool = True):
        """Preprocess, bin-sort and blend one image. sync_pairs=True reads the
        pair count back to the host (and returns it) and fails with GS_ERR_CAPACITY
        before sorting if it exceeds the capacity; sync_pairs=False keeps the count
        on the device (no synchronisation): check pairs_overflowed() afterwards."""
        g, app = scene.gaussians(), scene.appearance(self.kind, sh_degree)
        P = gs_preprocess(cam, g, app, self.pre, self.workspace, self.ws_bytes, stream, sync_pairs=sync_pairs)
        gs_bin_sort(cam, self.pre, self.n, P if sync_pairs else GS_PAIRS_ON_DEVICE, self.capacity, self.values,
                    self.tile_ids, self.ranges, self.workspace, self.ws_bytes, stream)
        gs_render_fwd(cam, self.pre, self.n, self.values, self.ranges, self.image, self.final_T, self.n_contrib,
                      stream)
        self.last_pairs = P
        return P

    def pairs_overflowed(self) -> bool:
        """After a device-mode forward: did the pair count exceed the capacity (synchronises)?"""
        return int(self.num_pairs.item()) > self.capacity

    def backward(self, cam: Camera, scene: SceneTensors, dL_dimage, sh_degree: int = 3, stream=None):
        g, app = scene.gaussians(), scene.appearance(self.kind, sh_degree)
        gs_render_bwd(cam, g, app, self.pre, self.values, self.ranges, self.final_T, self.n_contrib, dL_dimage,
                      self.grads, self.workspace, self.ws_bytes, stream)

    def splat_fields(self) -> dict:
        """Host copy of the splat records, split into fields."""
        raw = self.splats.view(-1, 16).cpu()
        f = raw.numpy()
        w = SPLAT_WORDS
        rect = raw.view(torch.int32).numpy()[:, w["rect"]:w["rect"] + 2]
        r01, r23 = rect[:, 0].astype("int64") & 0xFFFFFFFF, rect[:, 1].astype("int64") & 0xFFFFFFFF
        import numpy as np
        rects = np.stack([r01 & 0xFFFF, r01 >> 16, r23 & 0xFFFF, r23 >> 16]).astype(np.int32)
        return dict(mean2d=f[:, w["mean_x"]:w["mean_y"] + 1].T.copy(), conic=f[:, w["conic_a"]:w["conic_c"] + 1].T.copy(),
                    opacity=f[:, w["opacity"]].copy(), color=f[:, w["color"]:w["color"] + 3].T.copy(),
                    power_min=f[:, w["power_min"]].copy(), ext=f[:, w["ext_x"]:w["ext_y"] + 1].T.copy(),
                    depth=f[:, w["depth"]].copy(), rect=rects)
