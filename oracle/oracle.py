"""ctypes wrapper of the CPU oracle (gs_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by the test-suite, by the smoke check and by
the benchmark's CPU-baseline leg. It does not import the GPU package; scenes and
cameras are taken by attribute (any object with the fields of the seeded input
generator's Scene and Camera works).

Every function mirrors one stage of the method (the paper's Sec. 3.1 preprocess
and blend, Sec. 4 appearance models, and the fused backward of its appendix);
the arithmetic lives in C, this file only marshals arrays, apart from the
first-layer folding of the neural decoder (neural_fold), one matrix product in
numpy.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "_build", "libgsoracle.so")
_SOURCES = ("gs_oracle.c", "gs_oracle_body.inc", "gs_oracle.h")

APP_SH3 = 0
APP_LATENT_MLP = 1
APP_NEURAL = 2
APP_NEURAL_FOLDED = 3     # render only
APP_NASG = 4
APP_NASGABOR = 5
VISIBLE = 1
CLAMP_X = 2
CLAMP_Y = 4


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (no fast-math, no FMA contraction)."""
    os.makedirs(os.path.dirname(_LIB_PATH), exist_ok=True)
    if not force and os.path.exists(_LIB_PATH):
        lib_t = os.path.getmtime(_LIB_PATH)
        if all(os.path.getmtime(os.path.join(_HERE, s)) <= lib_t for s in _SOURCES):
            return _LIB_PATH
    tmp = _LIB_PATH + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
           "-shared", "-fPIC", "-o", tmp, os.path.join(_HERE, "gs_oracle.c"), "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class _Camera(C.Structure):
    _fields_ = [("viewmat", C.c_double * 12), ("campos", C.c_double * 3),
                ("fx", C.c_double), ("fy", C.c_double), ("cx", C.c_double), ("cy", C.c_double),
                ("width", C.c_int32), ("height", C.c_int32), ("near_plane", C.c_double),
                ("bg", C.c_double * 3)]


class _Appearance(C.Structure):
    _fields_ = [("kind", C.c_int32), ("sh_degree", C.c_int32), ("sh", C.c_void_p),
                ("latent", C.c_void_p), ("mlp_w", C.c_void_p), ("dir_exact", C.c_int32),
                ("half_act", C.c_int32), ("base_color", C.c_void_p), ("features", C.c_void_p),
                ("preact", C.c_void_p), ("lobes", C.c_void_p), ("sh_y0_folded", C.c_int32),
                ("neural_layers", C.c_int32), ("neural_width", C.c_int32), ("neural_raw16", C.c_int32)]


class _Pre(C.Structure):
    _fields_ = [("mean2d", C.c_void_p), ("conic", C.c_void_p), ("opacity", C.c_void_p),
                ("color", C.c_void_p), ("depth", C.c_void_p), ("rect", C.c_void_p),
                ("tiles", C.c_void_p), ("flags", C.c_void_p), ("mlp_mask", C.c_void_p)]


class _Grads(C.Structure):
    _fields_ = [(name, C.c_void_p) for name in (
        "dmeans", "dlog_scales", "dquats", "dopacity_logits", "dsh", "dlatent", "dmlp_w",
        "dmean2d", "dconic", "dopacity", "dcolor", "dbase_color", "dfeatures", "dlobes", "dmlp_w_abs")]


_lib = None


def lib():
    global _lib
    if _lib is None:
        _lib = C.CDLL(build())
        vp, i64 = C.c_void_p, C.c_int64
        for sfx in ("_f32", "_f64"):
            f = getattr(_lib, "orc_preprocess" + sfx)
            f.argtypes = [C.POINTER(_Camera), i64, vp, vp, vp, vp, C.POINTER(_Appearance), C.POINTER(_Pre)]
            f.restype = C.c_int
            f = getattr(_lib, "orc_render_fwd" + sfx)
            f.argtypes = [C.POINTER(_Camera), i64, C.POINTER(_Pre), vp, vp, vp, vp, vp, vp, vp, vp]
            f.restype = None
            f = getattr(_lib, "orc_render_bwd" + sfx)
            f.argtypes = [C.POINTER(_Camera), i64, vp, vp, vp, vp, C.POINTER(_Appearance), C.POINTER(_Pre),
                          vp, vp, vp, C.POINTER(_Grads)]
            f.restype = C.c_int
        _lib.orc_bin_sort.argtypes = [i64, vp, vp, vp, C.c_int32, C.c_int32, i64, vp, vp, vp]
        _lib.orc_bin_sort.restype = i64
        _lib.orc_sh_basis.argtypes = [vp, vp, vp]
        _lib.orc_sh_basis.restype = None
        _lib.orc_mlp_eval.argtypes = [vp, i64, vp, vp, C.c_int32]
        _lib.orc_mlp_eval.restype = None
        _lib.orc_round_half.argtypes = [C.c_double]
        _lib.orc_round_half.restype = C.c_double
        _lib.orc_lobe_eval_many.argtypes = [vp, C.c_int32, i64, vp, vp]
        _lib.orc_lobe_eval_many.restype = None
        _lib.orc_lobe_grad.argtypes = [vp, C.c_int32, vp, vp, vp]
        _lib.orc_lobe_grad.restype = C.c_double
    return _lib


def _p(a: np.ndarray | None):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def camera_struct(cam) -> _Camera:
    c = _Camera()
    vm = np.asarray(cam.viewmat, dtype=np.float64).reshape(-1)
    for k in range(12):
        c.viewmat[k] = vm[k]
    for k in range(3):
        c.campos[k] = float(cam.campos[k])
        c.bg[k] = float(cam.bg[k])
    c.fx, c.fy, c.cx, c.cy = float(cam.fx), float(cam.fy), float(cam.cx), float(cam.cy)
    c.width, c.height = int(cam.width), int(cam.height)
    c.near_plane = float(cam.near)
    return c


def half_to_f64(a: np.ndarray) -> np.ndarray:
    """binary16 bit patterns (uint16) to float64; float arrays pass through unchanged."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.float16)
    return np.ascontiguousarray(a.astype(np.float64))


class _SceneArrays:
    """float64 copies of a scene's arrays, kept alive while C reads them."""

    def __init__(self, scene, kind: int, sh_degree: int, dir_exact: bool = False, half_act: bool = False):
        self.n = int(scene.n)
        self.means = _f64(scene.means)
        self.log_scales = _f64(scene.log_scales)
        self.quats = _f64(scene.quats)
        self.opacity_logits = _f64(scene.opacity_logits)
        self.sh = _f64(scene.sh) if kind == APP_SH3 else None
        self.latent = half_to_f64(scene.latent) if kind == APP_LATENT_MLP else None
        neural = kind in (APP_NEURAL, APP_NEURAL_FOLDED)
        lobe = kind in (APP_NASG, APP_NASGABOR)
        self.mlp_w = (half_to_f64(scene.mlp_w) if kind == APP_LATENT_MLP else
                      half_to_f64(scene.neural_w) if neural else None)
        self.base_color = _f64(scene.base_color) if neural or lobe else None
        self.lobes = None
        if lobe:
            self.lobes = _f64(scene.lobes_gabor if kind == APP_NASGABOR else scene.lobes)
            assert self.lobes.shape[0] == (9 if kind == APP_NASGABOR else 8)
        self.features = half_to_f64(scene.features) if kind == APP_NEURAL else None
        # the folded form: pre-activations exact with exact inputs, else binary16 like its inputs
        self.preact = (np.ascontiguousarray(neural_fold(scene.features, scene.neural_w, exact=dir_exact))
                       if kind == APP_NEURAL_FOLDED else None)
        self.app = _Appearance(kind, sh_degree, _p(self.sh), _p(self.latent), _p(self.mlp_w), int(dir_exact),
                               int(half_act), _p(self.base_color), _p(self.features), _p(self.preact),
                               _p(self.lobes), int(bool(getattr(scene, "sh_y0_folded", False))),
                               *neural_arch(scene))


def neural_arch(scene) -> tuple:
    """(hidden layers, width, raw16) of a scene's neural decoder; the paper's default (2, 16, 0)."""
    arch = getattr(scene, "neural_arch", None)
    return tuple(int(v) for v in arch) if arch is not None else (2, 16, 0)


def neural_weight_count(layers: int, width: int) -> int:
    return 32 * width + (layers - 1) * width * width + 3 * width


def neural_fold(features, neural_w, exact: bool = False) -> np.ndarray:
    """First-layer folding of the neural decoder (the paper's viewer, supplementary
    section on the WebGL implementation): the inputs that do not depend on the
    view, x_0 = Y_0 and x_16..31 = (sin f_j, cos f_j), times their 17 columns of
    W1, as one pre-activation per hidden neuron and Gaussian, [16][n] float64.
    Unless ``exact``, the inputs are binary16 as the decoder sees them and the
    pre-activations are rounded to binary16, the precision they are stored in."""
    w1 = half_to_f64(neural_w)[: 16 * 32].reshape(16, 32)
    f = half_to_f64(features)
    enc = np.empty((16, f.shape[1]))
    enc[0::2] = np.sin(f)
    enc[1::2] = np.cos(f)
    y0 = 0.5 / np.sqrt(np.pi)
    if not exact:
        enc = enc.astype(np.float16).astype(np.float64)
        y0 = float(np.float16(y0))
    p = np.outer(w1[:, 0], np.full(f.shape[1], y0)) + w1[:, 16:] @ enc
    return p if exact else p.astype(np.float16).astype(np.float64)


def _kind_of(kind) -> int:
    if kind in ("sh3", APP_SH3):
        return APP_SH3
    if kind in ("latent", APP_LATENT_MLP):
        return APP_LATENT_MLP
    if kind in ("neural", APP_NEURAL):
        return APP_NEURAL
    if kind in ("neural_folded", APP_NEURAL_FOLDED):
        return APP_NEURAL_FOLDED
    if kind in ("nasg", APP_NASG):
        return APP_NASG
    if kind in ("nasgabor", APP_NASGABOR):
        return APP_NASGABOR
    raise ValueError(kind)


class Preprocessed(dict):
    """Planar preprocess outputs (float64 and int32 arrays) plus the C view of them."""

    def struct(self) -> _Pre:
        return _Pre(*[_p(self[k]) for k in ("mean2d", "conic", "opacity", "color", "depth", "rect",
                                             "tiles", "flags", "mlp_mask")])


def preprocess(cam, scene, kind="sh3", sh_degree: int = 3, mode: str = "f32",
               dir_exact: bool = False, half_act: bool = False) -> Preprocessed:
    kind = _kind_of(kind)
    sa = _SceneArrays(scene, kind, sh_degree, dir_exact, half_act)
    n = sa.n
    out = Preprocessed(
        mean2d=np.zeros((2, n)), conic=np.zeros((3, n)), opacity=np.zeros(n), color=np.zeros((3, n)),
        depth=np.zeros(n), rect=np.zeros((4, n), np.int32), tiles=np.zeros(n, np.int32),
        flags=np.zeros(n, np.int32), mlp_mask=np.zeros(n, np.uint64))
    st = out.struct()
    rc = getattr(lib(), "orc_preprocess_" + mode)(C.byref(camera_struct(cam)), n, _p(sa.means),
                                                   _p(sa.log_scales), _p(sa.quats), _p(sa.opacity_logits),
                                                   C.byref(sa.app), C.byref(st))
    if rc != 0:
        raise ValueError("oracle preprocess rejected its arguments")
    return out


def tile_grid(cam) -> tuple:
    return (int(cam.width) + 15) // 16, (int(cam.height) + 15) // 16


def bin_sort(cam, pre: Preprocessed):
    """Sorted pair list: (values, tile_of, ranges[T][2])."""
    tx, ty = tile_grid(cam)
    n = pre["tiles"].size
    total = int(pre["tiles"].astype(np.int64).sum())
    values = np.zeros(max(total, 1), np.int32)
    tile_of = np.zeros(max(total, 1), np.int32)
    ranges = np.zeros((tx * ty, 2), np.int64)
    got = lib().orc_bin_sort(n, _p(pre["rect"]), _p(pre["depth"]), _p(pre["tiles"]), tx, ty, total,
                             _p(values), _p(tile_of), _p(ranges))
    assert got == total
    return values[:total], tile_of[:total], ranges


def render_fwd(cam, pre: Preprocessed, ranges, values, mode: str = "f32", n_blended=None, n_walked=None):
    """(image[3][H][W], final_T[H][W], n_contrib[H][W], margin[H][W]); n_blended, if
    given (int32 [H][W]), receives each pixel's number of composited entries, and
    n_walked its number of visited entries (the stopping one included)."""
    W, H = int(cam.width), int(cam.height)
    image = np.zeros((3, H, W))
    final_T = np.zeros((H, W))
    n_contrib = np.zeros((H, W), np.int32)
    margin = np.zeros((H, W))
    ranges = np.ascontiguousarray(ranges, dtype=np.int64)
    values = np.ascontiguousarray(values, dtype=np.int32)
    st = pre.struct()
    getattr(lib(), "orc_render_fwd_" + mode)(C.byref(camera_struct(cam)), pre["tiles"].size, C.byref(st),
                                             _p(ranges), _p(values), _p(image), _p(final_T), _p(n_contrib),
                                             _p(margin), None if n_blended is None else _p(n_blended),
                                             None if n_walked is None else _p(n_walked))
    return image, final_T, n_contrib, margin


def render_bwd(cam, scene, pre: Preprocessed, ranges, values, dL_dimage, kind="sh3", sh_degree: int = 3,
               mode: str = "f32", dir_exact: bool = False, half_act: bool = False) -> dict:
    kind = _kind_of(kind)
    if kind == APP_NEURAL_FOLDED:
        raise ValueError("the folded neural form renders only; differentiate the unfolded one")
    sa = _SceneArrays(scene, kind, sh_degree, dir_exact, half_act)
    n = sa.n
    g = dict(dmeans=np.zeros((3, n)), dlog_scales=np.zeros((3, n)), dquats=np.zeros((4, n)),
             dopacity_logits=np.zeros(n),
             dsh=np.zeros((48, n)) if kind == APP_SH3 else None,
             dlatent=np.zeros((14, n)) if kind == APP_LATENT_MLP else None,
             dmlp_w=(np.zeros(1664) if kind == APP_LATENT_MLP else
                     np.zeros(neural_weight_count(*neural_arch(scene)[:2])) if kind == APP_NEURAL else None),
             dmean2d=np.zeros((2, n)), dconic=np.zeros((3, n)), dopacity=np.zeros(n), dcolor=np.zeros((3, n)),
             dbase_color=np.zeros((3, n)) if kind in (APP_NEURAL, APP_NASG, APP_NASGABOR) else None,
             dfeatures=np.zeros((16 if neural_arch(scene)[2] else 8, n)) if kind == APP_NEURAL else None,
             dlobes=np.zeros((9 if kind == APP_NASGABOR else 8, n)) if kind in (APP_NASG, APP_NASGABOR) else None)
    g["dmlp_w_abs"] = None if g["dmlp_w"] is None else np.zeros_like(g["dmlp_w"])
    gs = _Grads(*[_p(g[k]) for k in ("dmeans", "dlog_scales", "dquats", "dopacity_logits", "dsh", "dlatent",
                                      "dmlp_w", "dmean2d", "dconic", "dopacity", "dcolor", "dbase_color",
                                      "dfeatures", "dlobes", "dmlp_w_abs")])
    dimg = _f64(dL_dimage)
    ranges = np.ascontiguousarray(ranges, dtype=np.int64)
    values = np.ascontiguousarray(values, dtype=np.int32)
    st = pre.struct()
    rc = getattr(lib(), "orc_render_bwd_" + mode)(C.byref(camera_struct(cam)), n, _p(sa.means),
                                                   _p(sa.log_scales), _p(sa.quats), _p(sa.opacity_logits),
                                                   C.byref(sa.app), C.byref(st), _p(ranges), _p(values),
                                                   _p(dimg), C.byref(gs))
    if rc != 0:
        raise ValueError("oracle backward rejected its arguments")
    return {k: v for k, v in g.items() if v is not None}


def render(cam, scene, kind="sh3", sh_degree: int = 3, mode: str = "f32", dir_exact: bool = False,
           half_act: bool = False) -> dict:
    """All forward stages; returns a dict with the intermediate results."""
    pre = preprocess(cam, scene, kind, sh_degree, mode, dir_exact, half_act)
    values, tile_of, ranges = bin_sort(cam, pre)
    n_blended = np.zeros((int(cam.height), int(cam.width)), np.int32)
    n_walked = np.zeros((int(cam.height), int(cam.width)), np.int32)
    image, final_T, n_contrib, margin = render_fwd(cam, pre, ranges, values, mode, n_blended, n_walked)
    return dict(pre=pre, values=values, tile_of=tile_of, ranges=ranges, image=image, final_T=final_T,
                n_contrib=n_contrib, margin=margin, n_blended=n_blended, n_walked=n_walked)


def set_threads(k: int):
    """Threads of the oracle's parallel loops (its results do not depend on them)."""
    lib().orc_set_threads(int(k))


def get_threads() -> int:
    return int(lib().orc_get_threads())


def sh_basis(d) -> tuple:
    d = _f64(d)
    Y = np.zeros(16)
    dY = np.zeros(48)
    lib().orc_sh_basis(_p(d), _p(Y), _p(dY))
    return Y, dY.reshape(16, 3)


def mlp_eval(x, mlp_w, half_act: bool = False) -> np.ndarray:
    """Decoder colours [rows][3] of inputs x [rows][17] (binary16 bits or values)."""
    xx = half_to_f64(x).reshape(-1, 17)
    w = half_to_f64(mlp_w)
    out = np.zeros((xx.shape[0], 3))
    lib().orc_mlp_eval(_p(np.ascontiguousarray(xx)), xx.shape[0], _p(w), _p(out), int(half_act))
    return out


def lobe_eval(raw, gabor: bool, dirs) -> np.ndarray:
    """NASG (NASGabor) lobe kernel values at unit directions dirs [m][3] for the raw
    parameters raw[5] (raw[6]): frame angles, sharpness, anisotropy[, frequency]."""
    r = _f64(np.asarray(raw, np.float64).ravel())
    v = np.ascontiguousarray(np.asarray(dirs, np.float64).reshape(-1, 3))
    out = np.zeros(v.shape[0])
    lib().orc_lobe_eval_many(_p(r), int(gabor), v.shape[0], _p(v), _p(out))
    return out


def lobe_grad(raw, gabor: bool, d) -> tuple:
    """(G, dG/draw, dG/dd) of one lobe at one direction."""
    r = _f64(np.asarray(raw, np.float64).ravel())
    v = _f64(np.asarray(d, np.float64).ravel())
    dr = np.zeros(6)
    dv = np.zeros(3)
    G = lib().orc_lobe_grad(_p(r), int(gabor), _p(v), _p(dr), _p(dv))
    return G, dr[: 6 if gabor else 5], dv


def round_half(x: float) -> float:
    return lib().orc_round_half(float(x))
