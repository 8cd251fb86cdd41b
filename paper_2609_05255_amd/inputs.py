"""Seeded synthetic inputs for the rasterizer: scenes, cameras, upstream gradients.

This module only draws random numbers and builds pinhole cameras. It holds none
of the rasterizer's arithmetic (no projection, no appearance, no blending), so
both the GPU path and the CPU oracle can take their inputs from it.

The scenes stand in for the paper's trained real-world models (about 3M
Gaussians on Mip-NeRF 360, Sec. 4 and the densification table); every value is
drawn from the distributions listed in ``CONFIGS`` with numpy's PCG64.

Layouts (all planar, channel-major, C-contiguous numpy arrays):
  means          float32 [3][n]
  log_scales     float32 [3][n]
  quats          float32 [4][n]   (w, x, y, z), unit length as drawn
  opacity_logits float32 [n]
  sh             float32 [48][n]  row 3*k + c holds basis k, colour channel c
  latent         uint16  [14][n]  IEEE binary16 bit patterns
  mlp_w          uint16  [1664]   binary16 W1[32][17], W2[32][32], W3[3][32]
  base_color     float32 [3][n]   neural appearance: base colour c0
  features       uint16  [8][n]   neural appearance: binary16 features
  neural_w       uint16  [816]    binary16 W1[16][32], W2[16][16], W3[3][16]
  lobes          float32 [8][n]   NASG lobe: raw frame angles (3), raw sharpness,
                                  raw anisotropy, raw amplitudes (3)
  lobes_gabor    float32 [9][n]   NASGabor: the same rows, then the raw frequency
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

TILE = 16
SH_COEFFS = 48
LATENT_DIM = 14
MLP_IN = 17
MLP_HIDDEN = 32
MLP_OUT = 3
MLP_W_COUNT = MLP_HIDDEN * MLP_IN + MLP_HIDDEN * MLP_HIDDEN + MLP_OUT * MLP_HIDDEN  # 1664
NEURAL_FEATURES = 8
NEURAL_IN, NEURAL_HIDDEN = 32, 16
NEURAL_W_COUNT = NEURAL_HIDDEN * NEURAL_IN + NEURAL_HIDDEN * NEURAL_HIDDEN + MLP_OUT * NEURAL_HIDDEN  # 816
Y0 = 0.28209479177387814   # 1 / sqrt(4 pi), the degree-0 SH value

SCENE_SEED = 0
CAMERA_SEED_BASE = 1000
GRAD_SEED_BASE = 2000


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    n: int
    width: int
    height: int
    n_cameras: int
    means: str            # "uniform1" (U[-1,1]^3) or "normal0.6" (N(0, 0.6^2 I))
    log_scale_mu: float
    log_scale_sigma: float
    appearance: tuple     # subset of ("sh3", "latent", "neural", "nasg", "nasgabor")
    fixed_camera: bool = False


# The five workloads: tiny CPU-checkable, medium, paper-scale SH3, paper-scale
# latent+MLP (same geometry as the SH3 scene), large stress scene.
CONFIGS = {
    "tiny": Config("tiny", 1024, 64, 64, 1, "uniform1", -3.0, 0.3, ("sh3",), fixed_camera=True),
    "medium": Config("medium", 200_000, 1280, 720, 8, "normal0.6", -4.5, 0.5, ("sh3",)),
    "paper_sh3": Config("paper_sh3", 3_000_000, 1600, 1064, 16, "normal0.6", -5.0, 0.6, ("sh3",)),
    "paper_latent": Config("paper_latent", 3_000_000, 1600, 1064, 16, "normal0.6", -5.0, 0.6, ("latent",)),
    "stress": Config("stress", 6_000_000, 1920, 1080, 16, "normal0.6", -5.5, 0.7, ("sh3", "latent")),
    "paper_neural": Config("paper_neural", 3_000_000, 1600, 1064, 16, "normal0.6", -5.0, 0.6, ("neural",)),
    "paper_nasg": Config("paper_nasg", 3_000_000, 1600, 1064, 16, "normal0.6", -5.0, 0.6, ("nasg",)),
    "paper_nasgabor": Config("paper_nasgabor", 3_000_000, 1600, 1064, 16, "normal0.6", -5.0, 0.6, ("nasgabor",)),
}


def _rng(seed: int, stream: int) -> np.random.Generator:
    # One independent PCG64 stream per field, so adding a field never shifts another.
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream])))


@dataclasses.dataclass
class Scene:
    n: int
    means: np.ndarray
    log_scales: np.ndarray
    quats: np.ndarray
    opacity_logits: np.ndarray
    sh: np.ndarray | None = None
    latent: np.ndarray | None = None
    mlp_w: np.ndarray | None = None
    base_color: np.ndarray | None = None
    features: np.ndarray | None = None
    neural_w: np.ndarray | None = None
    lobes: np.ndarray | None = None
    lobes_gabor: np.ndarray | None = None
    neural_arch: tuple | None = None   # (hidden layers, width, raw16); None = the paper's (2, 16, 0)

    def subset(self, idx: np.ndarray) -> "Scene":
        idx = np.asarray(idx)
        pick = lambda a: None if a is None else np.ascontiguousarray(a[:, idx])
        copy = lambda a: None if a is None else a.copy()
        return Scene(len(idx), pick(self.means), pick(self.log_scales), pick(self.quats),
                     np.ascontiguousarray(self.opacity_logits[idx]), pick(self.sh), pick(self.latent),
                     copy(self.mlp_w), pick(self.base_color), pick(self.features), copy(self.neural_w),
                     pick(self.lobes), pick(self.lobes_gabor), self.neural_arch)


def make_scene(cfg: Config | str, seed: int = SCENE_SEED, n: int | None = None,
               appearance: tuple | None = None, neural_arch: tuple | None = None) -> Scene:
    """Draw a scene of ``cfg``'s distributions (``n`` overrides the count).
    ``neural_arch`` = (hidden layers 1..3, width 16 or 32, raw16) picks one of the
    neural decoder configurations of the paper's table (default (2, 16, 0)):
    raw16 stores 16 raw binary16 features instead of 8 frequency-encoded ones."""
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    n = cfg.n if n is None else int(n)
    appearance = cfg.appearance if appearance is None else appearance
    f32 = np.float32
    if cfg.means == "uniform1":
        means = _rng(seed, 1).uniform(-1.0, 1.0, size=(3, n)).astype(f32)
    else:
        means = (_rng(seed, 1).standard_normal((3, n), dtype=f32) * f32(0.6)).astype(f32)
    log_scales = (_rng(seed, 2).standard_normal((3, n), dtype=f32) * f32(cfg.log_scale_sigma)
                  + f32(cfg.log_scale_mu)).astype(f32)
    q = _rng(seed, 3).standard_normal((4, n), dtype=np.float64)
    q /= np.linalg.norm(q, axis=0, keepdims=True)   # uniform on S^3
    quats = q.astype(f32)
    opacity_logits = _rng(seed, 4).standard_normal(n, dtype=f32)
    scene = Scene(n, np.ascontiguousarray(means), np.ascontiguousarray(log_scales),
                  np.ascontiguousarray(quats), opacity_logits)
    if "sh3" in appearance:
        sh = (_rng(seed, 5).standard_normal((SH_COEFFS, n), dtype=f32) * f32(0.05)).astype(f32)
        sh[0:3] = (_rng(seed, 6).standard_normal((3, n), dtype=f32) * f32(0.2) + f32(0.5)).astype(f32)
        scene.sh = np.ascontiguousarray(sh)
    if "latent" in appearance:
        z = (_rng(seed, 7).standard_normal((LATENT_DIM, n), dtype=f32) * f32(0.5))
        scene.latent = np.ascontiguousarray(z.astype(np.float16).view(np.uint16))
        scene.mlp_w = make_mlp_weights(seed)
    if "nasg" in appearance or "nasgabor" in appearance:
        # base colour as for the neural model; lobe raw values: frame angles N(0, 1),
        # sharpness exp(N(1, 0.5)), anisotropy exp(N(-0.5, 0.7)), amplitudes N(0.5, 0.3)
        # (the reference initialises them at 0.5), frequency 20 (tanh(N(-1.5, 0.5)) + 1)
        dc = (_rng(seed, 6).standard_normal((3, n), dtype=f32) * f32(0.2) + f32(0.5)).astype(f32)
        scene.base_color = np.ascontiguousarray((dc * f32(Y0)).astype(f32))
        z = _rng(seed, 11).standard_normal((9, n), dtype=f32)
        mu = np.array([0, 0, 0, 1.0, -0.5, 0.5, 0.5, 0.5, -1.5], f32)[:, None]
        sd = np.array([1, 1, 1, 0.5, 0.7, 0.3, 0.3, 0.3, 0.5], f32)[:, None]
        lobes = (z * sd + mu).astype(f32)
        scene.lobes = np.ascontiguousarray(lobes[:8])
        scene.lobes_gabor = np.ascontiguousarray(lobes)
    if "neural" in appearance:
        # base colour: the SH3 scenes' degree-0 colour with Y0 folded in (c0 = Y0 sh_0);
        # features N(0, 1) in binary16; all three layers Glorot (a non-zero residual)
        dc = (_rng(seed, 6).standard_normal((3, n), dtype=f32) * f32(0.2) + f32(0.5)).astype(f32)
        scene.base_color = np.ascontiguousarray((dc * f32(Y0)).astype(f32))
        layers, width, raw16 = neural_arch if neural_arch is not None else (2, NEURAL_HIDDEN, 0)
        fe = _rng(seed, 9).standard_normal((16 if raw16 else NEURAL_FEATURES, n), dtype=f32)
        scene.features = np.ascontiguousarray(fe.astype(np.float16).view(np.uint16))
        scene.neural_w = make_neural_weights(seed, layers, width)
        scene.neural_arch = None if neural_arch is None else (int(layers), int(width), int(raw16))
    return scene


def make_mlp_weights(seed: int = SCENE_SEED) -> np.ndarray:
    """Glorot-uniform weights U(+-sqrt(6/(fan_in+fan_out))), drawn fp32, stored fp16."""
    rng = _rng(seed, 8)
    parts = []
    for fan_out, fan_in in ((MLP_HIDDEN, MLP_IN), (MLP_HIDDEN, MLP_HIDDEN), (MLP_OUT, MLP_HIDDEN)):
        lim = math.sqrt(6.0 / (fan_in + fan_out))
        parts.append(rng.uniform(-lim, lim, size=fan_out * fan_in).astype(np.float32))
    w = np.concatenate(parts).astype(np.float16).view(np.uint16)
    assert w.size == MLP_W_COUNT
    return np.ascontiguousarray(w)


def make_neural_weights(seed: int = SCENE_SEED, layers: int = 2, width: int = NEURAL_HIDDEN) -> np.ndarray:
    """Glorot-uniform weights of the 32 -> width (x layers) -> 3 decoder (default
    32 -> 16 -> 16 -> 3), drawn fp32, stored fp16: W1[width][32], layers - 1
    matrices [width][width], Wout[3][width]."""
    rng = _rng(seed, 10)
    shapes = [(width, NEURAL_IN)] + [(width, width)] * (layers - 1) + [(MLP_OUT, width)]
    parts = []
    for fan_out, fan_in in shapes:
        lim = math.sqrt(6.0 / (fan_in + fan_out))
        parts.append(rng.uniform(-lim, lim, size=fan_out * fan_in).astype(np.float32))
    w = np.concatenate(parts).astype(np.float16).view(np.uint16)
    assert w.size == NEURAL_IN * width + (layers - 1) * width * width + MLP_OUT * width
    return np.ascontiguousarray(w)


@dataclasses.dataclass
class Camera:
    viewmat: np.ndarray   # float32 [3][4] world -> camera (x right, y down, z forward)
    campos: np.ndarray    # float32 [3]
    fx: float
    fy: float
    cx: float
    cy: float
    width: int
    height: int
    near: float = 0.2
    bg: tuple = (0.0, 0.0, 0.0)


def look_at_camera(pos, width: int, height: int, fov_x_deg: float = 60.0,
                   target=(0.0, 0.0, 0.0), bg=(0.0, 0.0, 0.0)) -> Camera:
    """Pinhole camera at ``pos`` looking at ``target``; horizontal field of view."""
    pos = np.asarray(pos, dtype=np.float64)
    fwd = np.asarray(target, dtype=np.float64) - pos
    fwd /= np.linalg.norm(fwd)
    up = np.array([0.0, 1.0, 0.0]) if abs(fwd[1]) <= 0.99 else np.array([0.0, 0.0, 1.0])
    right = np.cross(-up, fwd)
    right /= np.linalg.norm(right)
    down = np.cross(fwd, right)
    rot = np.stack([right, down, fwd])            # rows: camera axes in world
    t = -rot @ pos
    viewmat = np.concatenate([rot, t[:, None]], axis=1).astype(np.float32)
    f = width / (2.0 * math.tan(math.radians(fov_x_deg) / 2.0))
    return Camera(viewmat, pos.astype(np.float32), float(np.float32(f)), float(np.float32(f)),
                  width / 2.0, height / 2.0, width, height, 0.2, tuple(bg))


def make_cameras(cfg: Config | str, count: int | None = None) -> list:
    """Cameras on the sphere of radius 3 looking at the origin (seed 1000+i)."""
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    count = cfg.n_cameras if count is None else count
    cams = []
    for i in range(count):
        if cfg.fixed_camera:
            pos = np.array([0.0, 0.0, -3.0])
        else:
            v = np.random.default_rng(CAMERA_SEED_BASE + i).standard_normal(3)
            pos = 3.0 * v / np.linalg.norm(v)
        cams.append(look_at_camera(pos, cfg.width, cfg.height))
    return cams


def make_upstream_grad(width: int, height: int, cam_index: int = 0, sigma: float = 1e-3) -> np.ndarray:
    """dL/dimage ~ N(0, sigma^2), float32 [3][H][W], seed 2000+i."""
    g = np.random.default_rng(GRAD_SEED_BASE + cam_index).standard_normal((3, height, width), dtype=np.float32)
    return np.ascontiguousarray(g * np.float32(sigma))
