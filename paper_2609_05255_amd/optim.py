"""Fused Adam over a scene's parameters: the optimiser step of the paper's
training pipeline (supplementary implementation details), one gs_adam_step
launch per iteration for every parameter tensor.

Learning rates per parameter channel (the row of the planar layout):
  * geometry as in 3D Gaussian Splatting: means 1.6e-4, log-scales 5e-3,
    rotations 1e-3, opacity logits 0.05;
  * SH3 (the paper's table of appearance learning rates): the degree-0 rows
    0.0025 -- the paper folds Y0 into the base colour and scales its rate by
    Y0 instead, the same step in colour space, which the Y0-folded form takes --
    and every other coefficient 0.000125;
  * latent + MLP: latents 0.008 (the paper's rate for the neural features) and
    decoder weights 0.003 with a second-moment decay of 0.99 (they receive a
    gradient from every visible Gaussian in every iteration);
  * neural (the paper's model): base colour 0.00025, features 0.008, decoder
    weights 0.003 with a second-moment decay of 0.99;
  * NASG / NASGabor: base colour 0.00025 and every lobe parameter
    0.0025 (0.3536 / dbar)^2, dbar the mean distance from each training camera
    to its three nearest neighbours (camera_spacing).
The latents and the decoder weights have fp32 master copies here; each step
writes their binary16 copies into the scene buffers the passes read, as the
paper does for its decoder weights.
"""
from __future__ import annotations

import torch

from . import gsraster as gs

LR_MEANS, LR_SCALES, LR_QUATS, LR_OPACITY = 1.6e-4, 5e-3, 1e-3, 0.05
LR_SH_DC, LR_SH_REST = 0.0025, 0.000125
Y0 = 0.28209479177387814   # 1 / (2 sqrt(pi)), the degree-0 SH value
LR_LATENT, LR_MLP, BETA2_MLP = 0.008, 0.003, 0.99
LR_BASE_COLOR, LR_FEATURES = 0.00025, 0.008
LR_LOBES, LOBE_SPACING_REF = 0.0025, 0.3536
NEURAL_FEATURES = 8
LATENT_DIM = 14


def camera_spacing(campos) -> float:
    """Mean over the training cameras of the mean distance to their three nearest neighbours."""
    c = torch.as_tensor(campos, dtype=torch.float64).reshape(-1, 3)
    dist = torch.cdist(c, c)
    dist.fill_diagonal_(float("inf"))
    k = min(3, c.shape[0] - 1)
    return float(dist.topk(k, dim=1, largest=False).values.mean()) if k > 0 else LOBE_SPACING_REF


class FusedAdam:
    def __init__(self, scene: gs.SceneTensors, frame: gs.Frame, kind: int, betas=(0.9, 0.999), eps: float = 1e-15,
                 camera_dbar: float = LOBE_SPACING_REF):
        self.beta1, self.beta2, self.eps, self.t = betas[0], betas[1], eps, 0
        self.kind = kind
        self.groups = []

        def add(param, grad, lr_rows, beta2=None, half=None):
            rows = len(lr_rows)
            param = param.view(rows, -1)
            assert param.is_contiguous() and grad.numel() == param.numel()
            self.groups.append(dict(param=param, grad=grad, exp_avg=torch.zeros_like(param),
                                    exp_avg_sq=torch.zeros_like(param), param_half=half, rows=rows,
                                    n=param.shape[1], beta2=self.beta2 if beta2 is None else beta2,
                                    lr=list(lr_rows)))

        add(scene.means, frame.dmeans, [LR_MEANS] * 3)
        add(scene.log_scales, frame.dlog_scales, [LR_SCALES] * 3)
        add(scene.quats, frame.dquats, [LR_QUATS] * 4)
        add(scene.opacity_logits, frame.dopacity_logits, [LR_OPACITY])
        if kind == gs.GS_APP_SH3:
            lr_dc = LR_SH_DC * Y0 if scene.sh_y0_folded else LR_SH_DC
            add(scene.sh, frame.dsh, [lr_dc] * 3 + [LR_SH_REST] * 45)
        elif kind in gs.LOBE_ROWS:
            lobes = scene.lobes_gabor if kind == gs.GS_APP_NASGABOR else scene.lobes
            lr_lobe = LR_LOBES * (LOBE_SPACING_REF / camera_dbar) ** 2
            add(scene.base_color, frame.dbase_color, [LR_BASE_COLOR] * 3)
            add(lobes, frame.dlobes, [lr_lobe] * gs.LOBE_ROWS[kind])
        elif kind == gs.GS_APP_NEURAL:
            self.features32 = scene.features.view(torch.float16).float().contiguous()
            self.mlp32 = scene.neural_w.view(torch.float16).float().contiguous()
            add(scene.base_color, frame.dbase_color, [LR_BASE_COLOR] * 3)
            add(self.features32, frame.dfeatures, [LR_FEATURES] * scene.features.shape[0], half=scene.features)
            add(self.mlp32, frame.dmlp_w, [LR_MLP], beta2=BETA2_MLP, half=scene.neural_w)
        else:
            self.latent32 = scene.latent.view(torch.float16).float().contiguous()
            self.mlp32 = scene.mlp_w.view(torch.float16).float().contiguous()
            add(self.latent32, frame.dlatent, [LR_LATENT] * LATENT_DIM, half=scene.latent)
            add(self.mlp32, frame.dmlp_w, [LR_MLP], beta2=BETA2_MLP, half=scene.mlp_w)

    def step(self, stream=None):
        self.t += 1
        gs.gs_adam_step(self.groups, self.beta1, self.eps, self.t, stream)

    def backward_step(self, frame: gs.Frame, cam: gs.Camera, scene: gs.SceneTensors, dL_dimage, sh_degree: int = 3,
                      grads: gs.Grads | None = None, stream=None):
        """The backward with this optimiser's step of the Gaussians' own parameters applied
        inside it (gs_render_bwd_adam, SH3): the same result as frame.backward then step(),
        without writing the gradients (pass `grads` to have them written as well)."""
        if self.kind != gs.GS_APP_SH3:
            raise ValueError("the step inside the backward is built for the SH3 appearance")
        self.t += 1
        g = grads if grads is not None else gs.Grads()
        gs.gs_render_bwd_adam(cam, scene.gaussians(), scene.appearance(self.kind, sh_degree), frame.pre,
                              frame.values, frame.ranges, frame.final_T, frame.n_contrib, dL_dimage, g,
                              self.groups[:gs.GS_RENDER_ADAM_TENSORS], self.beta1, self.eps, self.t, frame.workspace,
                              frame.ws_bytes, stream)

    def bytes_per_backward_step(self) -> int:
        """HBM bytes of the parameter update inside the backward (backward_step), beyond those
        the backward reads anyway: m and v read, param, m and v written, per element, and the
        parameters the backward itself does not read (culled Gaussians', inactive bands')."""
        total = 0
        for g in self.groups[:gs.GS_RENDER_ADAM_TENSORS]:
            total += g["rows"] * g["n"] * 5 * 4
        return total

    def bytes_per_step(self) -> int:
        """HBM bytes one step must move: per element param, grad, m and v read, param, m and v
        written (fp32), plus the binary16 copy where there is one."""
        total = 0
        for g in self.groups:
            e = g["rows"] * g["n"]
            total += e * (7 * 4 + (2 if g["param_half"] is not None else 0))
        return total
