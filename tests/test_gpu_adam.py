"""GPU parity of the fused Adam step (gs_adam_step through the C ABI) with the
float64 oracle of Algorithm 1 (oracle/adam.py). Each step is checked from the
GPU's own fp32 state of the previous step, so the bound is one step's fp32
rounding: moments within 4 ulp of their terms, parameters within 2 ulp plus
2e-6 of the update; the binary16 copy is bit-exact against the fp32 result
rounded to nearest even."""
import numpy as np
import pytest
import torch

from oracle import adam
from paper_2609_05255_amd import gsraster as gs
from parity import say

pytestmark = pytest.mark.gpu

B1, EPS = 0.9, 1e-8
U = 2.0 ** -23


def make_tensor(rng, rows, n, beta2, half, lr_scale):
    p = rng.normal(size=(rows, n)).astype(np.float32)
    t = dict(rows=rows, n=n, beta2=beta2, lr=list(lr_scale * rng.random(rows) + 1e-4),
             host_p=p, param=torch.from_numpy(p).cuda(),
             exp_avg=torch.zeros(rows, n, device="cuda"), exp_avg_sq=torch.zeros(rows, n, device="cuda"),
             grad=torch.zeros(rows, n, device="cuda"))
    if half:
        t["param_half"] = torch.zeros(rows, n, dtype=torch.int16, device="cuda")
    return t


def run_and_check(tensors, steps, rng, label):
    say("case adam %s: %s" % (label, ", ".join("%dx%d" % (t["rows"], t["n"]) for t in tensors)))
    for step in range(1, steps + 1):
        before = []
        for t in tensors:
            g = (rng.normal(size=(t["rows"], t["n"])) * np.exp(rng.normal(size=(t["rows"], 1)) * 3)).astype(np.float32)
            if t["n"] > 2:
                g[:, 1] = 0.0       # untouched element: the moments still decay
            t["grad"].copy_(torch.from_numpy(g))
            before.append((t["param"].cpu().numpy().astype(np.float64), g.astype(np.float64),
                           t["exp_avg"].cpu().numpy().astype(np.float64),
                           t["exp_avg_sq"].cpu().numpy().astype(np.float64)))
        gs.gs_adam_step(tensors, B1, EPS, step)
        torch.cuda.synchronize()
        for t, (p0, g, m0, v0) in zip(tensors, before):
            if t["n"] == 0:
                continue
            # the library receives its rates and decays as fp32 values: the oracle takes the same values
            f32 = lambda x: np.float64(np.float32(x))
            lr32 = np.asarray(t["lr"], np.float32).astype(np.float64)
            p_ref, m_ref, v_ref = adam.adam_step(p0, g, m0, v0, lr32, f32(B1), f32(t["beta2"]), f32(EPS), step)
            p = t["param"].cpu().numpy().astype(np.float64)
            m = t["exp_avg"].cpu().numpy().astype(np.float64)
            v = t["exp_avg_sq"].cpu().numpy().astype(np.float64)
            tol_m = 4 * U * (B1 * np.abs(m0) + (1 - B1) * np.abs(g)) + 1e-38
            tol_v = 4 * U * (t["beta2"] * v0 + (1 - t["beta2"]) * g * g) + 1e-38
            tol_p = 2 * U * np.abs(p_ref) + 2e-6 * np.abs(p_ref - p0) + 1e-38
            assert np.all(np.abs(m - m_ref) <= tol_m), (label, step, "m", float(np.max(np.abs(m - m_ref) / tol_m)))
            assert np.all(np.abs(v - v_ref) <= tol_v), (label, step, "v", float(np.max(np.abs(v - v_ref) / tol_v)))
            assert np.all(np.abs(p - p_ref) <= tol_p), (label, step, "p", float(np.max(np.abs(p - p_ref) / tol_p)))
            if "param_half" in t:
                h = t["param_half"].cpu().numpy().view(np.uint16)
                assert np.array_equal(h, adam.half_copy(p.astype(np.float32))), (label, step)
    say("  %d steps OK" % steps)


def test_adam_several_tensors_and_steps():
    rng = np.random.default_rng(10)
    ts = [make_tensor(rng, 3, 100_003, 0.999, False, 1e-3),     # means-like, ragged length
          make_tensor(rng, 48, 2_049, 0.999, False, 1e-4),      # SH-like, 48 rows
          make_tensor(rng, 14, 1_025, 0.999, True, 8e-3),       # latent master + half copy
          make_tensor(rng, 1, 1_664, 0.99, True, 3e-3),         # decoder weights, beta2 0.99
          make_tensor(rng, 4, 100_000, 0.999, True, 1e-3)]      # rows 16-byte aligned: vector accesses
    run_and_check(ts, 3, rng, "five tensors")


def test_adam_edge_sizes():
    rng = np.random.default_rng(11)
    ts = [make_tensor(rng, 2, 0, 0.999, False, 1e-3),
          make_tensor(rng, 1, 1, 0.999, True, 1e-2),
          make_tensor(rng, 5, 1_023, 0.9, False, 1e-3),
          make_tensor(rng, 5, 1_024, 0.999, True, 1e-3),
          make_tensor(rng, 60, 7, 0.999, False, 1e-3)]
    run_and_check(ts, 2, rng, "edge sizes")


@pytest.mark.parametrize("kind", ["latent", "neural", "neural_32", "nasgabor", "sh3_y0_folded"])
def test_fused_adam_on_a_scene(kind):
    # one training iteration on a tiny scene: the half-precision buffers the
    # passes read are the rounded fp32 masters, and every parameter moved by at
    # most its learning rate (|m_hat| / sqrt(v_hat) = 1 in a first step)
    from paper_2609_05255_amd import inputs
    from paper_2609_05255_amd.optim import FusedAdam
    from parity import tiny_camera
    kid = {"latent": gs.GS_APP_LATENT_MLP, "neural": gs.GS_APP_NEURAL, "neural_32": gs.GS_APP_NEURAL,
           "nasgabor": gs.GS_APP_NASGABOR, "sh3_y0_folded": gs.GS_APP_SH3}[kind]
    arch = (2, 32, 0) if kind == "neural_32" else None
    base = {"sh3_y0_folded": "sh3", "neural_32": "neural"}.get(kind, kind)
    sc = inputs.make_scene("tiny", appearance=(base,), neural_arch=arch)
    if kind == "sh3_y0_folded":
        sc.sh = sc.sh.copy()
        sc.sh[0:3] *= np.float32(0.28209479177387814)
        sc.sh_y0_folded = True
    cam = tiny_camera()
    st = gs.SceneTensors(sc)
    fr = gs.Frame(sc.n, cam.width, cam.height, kid, 1 << 16, neural_arch=arch)
    cs = gs.camera_struct(cam)
    fr.forward(cs, st)
    fr.backward(cs, st, torch.from_numpy(inputs.make_upstream_grad(cam.width, cam.height, 0)).cuda())
    opt = FusedAdam(st, fr, kid, camera_dbar=0.5)
    if kind == "sh3_y0_folded":   # the DC rows take the paper's rate 0.0025 Y0
        assert abs(opt.groups[4]["lr"][0] - 0.0025 * 0.28209479177387814) < 1e-12
    if kind == "nasgabor":        # lobe rows 0.0025 (0.3536 / dbar)^2
        assert abs(opt.groups[5]["lr"][0] - 0.0025 * (0.3536 / 0.5) ** 2) < 1e-12 and opt.groups[5]["rows"] == 9
    if kind == "neural_32":       # the 32-32-32-3 decoder's 2,144 weights in one group
        assert any(g["rows"] == 1 and g["param"].numel() == 2144 for g in opt.groups)
    before = [g["param"].clone() for g in opt.groups]
    opt.step()
    torch.cuda.synchronize()
    for g, b in zip(opt.groups, before):
        lr = torch.tensor(g["lr"], device="cuda").view(-1, 1)
        # (plus the fp32 rounding of the updated value)
        assert torch.all((g["param"] - b).abs() <= lr * (1 + 1e-5) + 2 * U * b.abs()), g["rows"]
        if g["param_half"] is not None:
            h = g["param_half"].view(g["rows"], -1).cpu().numpy().view(np.uint16)
            assert np.array_equal(h, adam.half_copy(g["param"].cpu().numpy()))
    say("  fused Adam on the %s scene: %d tensors, %d bytes per step" % (kind, len(opt.groups), opt.bytes_per_step()))


GRAD_NAMES = ("dmeans", "dlog_scales", "dquats", "dopacity_logits", "dsh")


@pytest.mark.parametrize("scene,sh_degree", [("tiny", 3), ("tiny", 1), ("medium", 3)])
def test_adam_inside_the_backward(scene, sh_degree):
    # gs_render_bwd_adam: the SH3 backward with the Adam step of the Gaussians'
    # own parameters applied where each gradient is computed, against
    # gs_render_bwd and then gs_adam_step. The gradients it also writes are the
    # backward's (up to the float atomics' summation order); the parameters and
    # moments it leaves are bit-exact against gs_adam_step applied to those very
    # gradients, culled Gaussians' and inactive bands' elements included.
    from paper_2609_05255_amd import inputs
    from paper_2609_05255_amd.optim import FusedAdam
    from parity import tiny_camera
    sc = inputs.make_scene(scene)
    cam = tiny_camera() if scene == "tiny" else inputs.make_cameras("medium")[4]
    say("case adam inside the backward: %s, degree %d, n=%d" % (scene, sh_degree, sc.n))
    st = gs.SceneTensors(sc)
    fr = gs.Frame(sc.n, cam.width, cam.height, gs.GS_APP_SH3, 1 << 22)
    cs = gs.camera_struct(cam)
    fr.forward(cs, st, sh_degree)
    up = torch.from_numpy(inputs.make_upstream_grad(cam.width, cam.height, 2)).cuda()
    fr.backward(cs, st, up, sh_degree)
    plain = {k: getattr(fr, k).clone() for k in GRAD_NAMES}
    opt = FusedAdam(st, fr, gs.GS_APP_SH3)
    gen = torch.Generator(device="cuda").manual_seed(5)
    for g in opt.groups:   # a moment history, as after a few steps
        g["exp_avg"].copy_(torch.randn(g["exp_avg"].shape, device="cuda", generator=gen) * 1e-3)
        g["exp_avg_sq"].copy_(torch.randn(g["exp_avg_sq"].shape, device="cuda", generator=gen).square() * 1e-6)
    opt.t = 4
    before = [(g["param"].clone(), g["exp_avg"].clone(), g["exp_avg_sq"].clone()) for g in opt.groups]
    for k in GRAD_NAMES:
        getattr(fr, k).fill_(float("nan"))
    opt.backward_step(fr, cs, st, up, sh_degree, grads=fr.grads)
    torch.cuda.synchronize()
    assert opt.t == 5
    for k in GRAD_NAMES:
        a, b = getattr(fr, k), plain[k]
        assert not torch.isnan(a).any(), k
        scale = float(b.abs().max())
        assert bool(((a - b).abs() <= 1e-4 * b.abs() + 1e-6 * scale).all()), (k, float((a - b).abs().max()))
    ref = []
    for g, (p0, m0, v0), k in zip(opt.groups, before, GRAD_NAMES):
        ref.append(dict(param=p0.clone(), grad=getattr(fr, k).view(g["rows"], -1), exp_avg=m0.clone(),
                        exp_avg_sq=v0.clone(), rows=g["rows"], n=g["n"], beta2=g["beta2"], lr=g["lr"]))
    gs.gs_adam_step(ref, opt.beta1, opt.eps, opt.t)
    torch.cuda.synchronize()
    for g, r in zip(opt.groups, ref):
        for key in ("param", "exp_avg", "exp_avg_sq"):
            assert torch.equal(g[key], r[key]), (g["rows"], key)
    # without gradient outputs the update is the same. Compared bit-exact for an
    # upstream gradient on one pixel: then no accumulator takes two float atomics,
    # and both calls see the same gradients.
    one = torch.zeros_like(up)
    one[:, cam.height // 2, cam.width // 2] = up[:, cam.height // 2, cam.width // 2]
    results = []
    for grads in (fr.grads, None):
        for g, (p0, m0, v0) in zip(opt.groups, before):
            g["param"].copy_(p0)
            g["exp_avg"].copy_(m0)
            g["exp_avg_sq"].copy_(v0)
        opt.t = 4
        opt.backward_step(fr, cs, st, one, sh_degree, grads=grads)
        torch.cuda.synchronize()
        results.append([(g["param"].clone(), g["exp_avg"].clone(), g["exp_avg_sq"].clone()) for g in opt.groups])
    moved = sum(int((x[0] != b[0]).sum()) for x, b in zip(results[1], before))
    for x, y in zip(*results):
        for u, w in zip(x, y):
            assert torch.equal(u, w)
    say("  bit-exact against the backward then gs_adam_step (%d elements); without gradient outputs the "
        "same bits (%d parameters moved)" % (sum(g["rows"] * g["n"] for g in opt.groups), moved))
