"""Benchmark of the rasterizer's forward + backward on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config paper_sh3]
                    [--no-cpu-baseline] [--no-extra]

One step = one full pass of the hot path for one camera of the scene:
gs_preprocess, gs_bin_sort (the pair count stays on the device: no host
synchronisation inside a step), gs_render_fwd and gs_render_bwd, cycling over
the configuration's cameras. Scene parameters and upstream gradients are
resident on the GPU before timing starts. Prints one JSON line: fwd+bwd
iterations/s of the headline workload (3M Gaussians, 1600x1064, SH3) and its
Mpix/s, per-kernel times measured with HIP events on the rendering stream, the
roofline of the dominant kernel, forward-only (render) rates, a training step
with the fused Adam update, and the CPU oracle timed on a bounded sample. The
same run measures the latent appearance on the same geometry (the paper's
compact-appearance comparison) and the stress workload (6M Gaussians,
1920x1080) with both appearances, per stage; --no-extra skips them.
"""
from __future__ import annotations

import argparse
import gc
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "fwd+bwd iterations/sec and rendered Mpix/s at 3M Gaussians, 1600x1064"
HBM_PEAK_GBS = 8000.0            # MI355X HBM3E
FP32_VECTOR_PEAK_TFLOPS = 157.3  # published; counts packed-fp32 FMA
FP32_UNPACKED_PEAK_TFLOPS = 78.6 # 256 CU x 4 SIMD x 16 lanes x 2 flops x 2.4 GHz (the kernels emit no packed fp32)
# fp32 work of the blend per (pixel, list entry), counting an FMA as 2, by what
# the method does with the entry. The method visits, per pixel, every entry up
# to the one that stops the pixel (forward) or up to its last contributor
# (backward); gs_render_work counts them ("walked_fwd", "listed"):
#   blended:   forward 24 (quadratic form 11, exp 2, alpha 2, transmittance 2,
#              weight 1, colour 6); backward 62 (quadratic form 11, exp 2, alpha 2,
#              transmittance 2, dcolour 4, dalpha 15, suffix sum 6, dopacity and
#              the dL/dpower moments 20)
#   visited but not blended (power > 0, alpha below 1/255, or the stopping
#   entry): 15 (quadratic form 11, exp 2, alpha 2) in either direction. The
#   kernels skip part of these for a whole tile with a conservative box test;
#   the work counted is the method's, not what remains after that skip.
BLEND_FLOPS = {"blend_fwd": (24.0, 15.0), "blend_bwd": (62.0, 15.0)}
STAGES = {"preprocess": ("preprocess", "pair_count"),
          "sort": ("depth_sort", "entry_offsets", "block_entries", "block_sort", "tile_lists"),
          "blend": ("blend_fwd",),
          "backward": ("bwd_prep", "blend_bwd", "preprocess_bwd", "mlp_reduce")}


# HBM traffic of a kernel, from memory-counter runs summarised under profiles/
# (FETCH_SIZE and WRITE_SIZE per dispatch, each scaled by what the counter reads
# for a copy of known size). Each summary records a hash of the kernel's
# sources and of the build script (its per-file compiler options); once they
# change, the recorded figure no longer describes the kernel and the traffic is
# reported as null.
TRAFFIC_SUMMARIES = {("blend_bwd", "paper_sh3", "sh3"): "profiles/blend_bwd_paper_sh3_traffic.txt"}
KERNEL_SOURCES = {"blend_bwd": ("paper_2609_05255_amd/csrc/blend.hip", "paper_2609_05255_amd/csrc/gs_internal.h",
                                 "paper_2609_05255_amd/build.py")}


def source_hash(kernel: str) -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def recorded_traffic(kernel: str, config: str, kind: str) -> float | None:
    """Bytes per launch from the committed counter summary, or None."""
    rel = TRAFFIC_SUMMARIES.get((kernel, config, kind))
    if rel is None or not os.path.exists(os.path.join(ROOT, rel)):
        return None
    fields = {}
    with open(os.path.join(ROOT, rel)) as f:
        for line in f:
            if ":" in line and not line.startswith(" "):
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
    if fields.get("source_hash") != source_hash(kernel):
        return None
    try:
        return float(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=32)
    ap.add_argument("--warmup", type=int, default=4)
    ap.add_argument("--config", default="paper_sh3")
    ap.add_argument("--appearance", default=None,
                    help="sh3, latent, neural, nasg or nasgabor (default: the config's first)")
    ap.add_argument("--neural-arch", default=None,
                    help="neural decoder as 'layers,width,raw16' (the paper's configurations table; "
                         "default 2,16,0)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="measure only --config (not the latent and stress comparisons)")
    ap.add_argument("--copy-probe-mb", type=int, default=0,
                    help="before the steps, one device-to-device copy of this many MB (a plain copy kernel of "
                         "known size, to calibrate memory-traffic counters)")
    return ap.parse_args()


def appearance_bytes(kind: str, sh_degree: int = 3) -> int:
    """Appearance bytes per visible Gaussian: SH3 48 fp32, latent 14 binary16, neural a 12 B base
    colour and 8 binary16 features (the folded form: the base colour and 16 binary16
    pre-activations, 44 B; NASG 12 + 32 B, NASGabor 12 + 36 B; 16 raw binary16 features: 12 + 32 B)."""
    if kind == "sh3":
        return 4 * 3 * (sh_degree + 1) ** 2
    return {"neural_folded": 44, "neural_raw16": 44, "nasg": 44, "nasgabor": 48}.get(kind, 28)


def algorithmic_bytes(kernel: str, n: int, vis: float, kind: str, pairs: float = 0.0, sh_degree: int = 3):
    """HBM bytes a launch (or stage) must move at minimum, averaged over cameras."""
    app = appearance_bytes(kind, sh_degree)
    # SH3 hands the backward the colour's 40-byte direction Jacobian (9 floats and the clamp bits)
    # in place of a second read of the coefficients
    jac = 40 if kind == "sh3" else 0
    if kernel == "preprocess":
        # params 44 B + tiles 4 B + depth key 4 B per Gaussian; appearance + 48 B of projected splat
        # (mean 8, conic 12, opacity 4, colour 12, rectangle 8, depth 4) + the Jacobian per visible
        # one; the record written is 64 B, the rest being the blend's early-skip fields
        return n * (44 + 8) + vis * (app + 48 + jac)
    if kernel == "preprocess_bwd":
        # tiles 4 B + dense gradient writes per Gaussian; params, accumulators and appearance (SH3:
        # its Jacobian) per visible one
        grad = 44 + 4 * {"sh3": 48, "latent": 14, "neural": 11, "neural_raw16": 19, "nasg": 11, "nasgabor": 12}[kind]
        return n * (4 + grad) + vis * (44 + 36 + (jac or app))
    if kernel == "bin_sort":
        # scan and pair emission: 8 B per Gaussian (tiles, offset), 16 B per visible one (rectangle,
        # depth, index), 12 B per pair written; the sort's lower bound: one read and one write of
        # every 12-byte pair
        return 8 * n + 16 * vis + 12 * pairs + 24 * pairs
    return None


def group_stages(stage_ms: dict) -> dict:
    return {g: round(sum(stage_ms.get(k, 0.0) for k in ks), 4) for g, ks in STAGES.items()}


def measure(gs, inputs, torch, cfg_name: str, kind: str, args, arch=None, train=True, render=True):
    """Times the fwd+bwd step of one workload; returns its figures (and, for
    the CPU baseline, its scene and cameras)."""
    cfg = inputs.CONFIGS[cfg_name]
    kid = {"sh3": gs.GS_APP_SH3, "latent": gs.GS_APP_LATENT_MLP, "neural": gs.GS_APP_NEURAL,
           "nasg": gs.GS_APP_NASG, "nasgabor": gs.GS_APP_NASGABOR}[kind]
    dev = "cuda:0"
    t0 = time.time()
    scene = inputs.make_scene(cfg, appearance=(kind,), neural_arch=arch)
    cams = inputs.make_cameras(cfg)
    st = gs.SceneTensors(scene, device=dev)
    grads_up = [torch.from_numpy(inputs.make_upstream_grad(cfg.width, cfg.height, i)).to(dev)
                for i in range(len(cams))]
    cstructs = [gs.camera_struct(c) for c in cams]
    print("# scene %s (%s) generated and uploaded in %.1fs" % (cfg.name, kind, time.time() - t0), file=sys.stderr,
          flush=True)
    if args.copy_probe_mb > 0:
        nbytes = args.copy_probe_mb << 20
        src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # size the pair buffers: preprocess every camera once (untimed, read back)
    probe = gs.Frame(scene.n, cfg.width, cfg.height, kid, 1, device=dev, neural_arch=arch)
    g, app = st.gaussians(), st.appearance(kid)
    pairs, visible = [], []
    for c in cstructs:
        pairs.append(gs.gs_preprocess(c, g, app, probe.pre, probe.workspace, probe.ws_bytes))
        visible.append(int((probe.tiles_touched[: scene.n] > 0).sum().item()))
    del probe
    capacity = int(max(pairs) * 1.02) + 4096
    fr = gs.Frame(scene.n, cfg.width, cfg.height, kid, capacity, device=dev, neural_arch=arch)
    stream = torch.cuda.current_stream()
    ncam = len(cstructs)

    def step(i):
        # the pair count stays on the device: no host synchronisation inside a step
        c = cstructs[i % ncam]
        fr.forward(c, st, stream=stream, sync_pairs=False)
        fr.backward(c, st, grads_up[i % ncam], stream=stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    assert not fr.pairs_overflowed(), "pair capacity exceeded"
    it_s = args.steps / elapsed

    # per-step spread: the same K steps again, a pair of events around each
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for i in range(args.steps):
        ev[i][0].record(stream)
        step(i)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    step_times = np.array([a.elapsed_time(b) for a, b in ev])

    # the blend's work per image (gs_render_work), over the cameras the steps visit
    steps_cams = [i % ncam for i in range(args.steps)]
    counts = torch.zeros(5, dtype=torch.int64, device=dev)
    work = {}
    for i in sorted(set(steps_cams)):
        fr.forward(cstructs[i], st, stream=stream, sync_pairs=False)
        gs.gs_render_work(cstructs[i], fr.pre, scene.n, fr.values, fr.ranges, counts, stream)
        work[i] = counts.cpu().numpy().astype(np.float64)
    w = np.mean([work[i] for i in steps_cams], axis=0)
    work_avg = {"blended": int(w[0]), "listed": int(w[1]), "evaluated_bwd": int(w[2]), "evaluated_fwd": int(w[3]),
                "walked_fwd": int(w[4])}

    # per-kernel durations: the same K steps again with HIP events around every kernel
    timer = gs.Timer()
    timer.attach()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    kt = timer.read()
    stage_ms = {k: (ms / cnt if cnt else 0.0) for k, (ms, cnt) in kt.items() if cnt}
    gs.Timer.detach()

    vis_avg = float(np.mean([visible[i] for i in steps_cams]))
    pairs_avg = float(np.mean([pairs[i] for i in steps_cams]))
    bkind = "neural_raw16" if kind == "neural" and arch and arch[2] else kind
    hbm = {}
    for k in ("preprocess", "preprocess_bwd"):
        if stage_ms.get(k, 0) > 0:
            b = algorithmic_bytes(k, scene.n, vis_avg, bkind)
            ach = b / (stage_ms[k] * 1e-3) / 1e9
            hbm[k] = {"algorithmic_MB": round(b / 1e6, 1), "ms": round(stage_ms[k], 4), "GB_s": round(ach, 1),
                      "frac": round(ach / HBM_PEAK_GBS, 4)}
    sort_ms = sum(stage_ms.get(k, 0.0) for k in STAGES["sort"])
    b = algorithmic_bytes("bin_sort", scene.n, vis_avg, bkind, pairs_avg)
    hbm["bin_sort"] = {"algorithmic_MB": round(b / 1e6, 1), "ms": round(sort_ms, 4),
                       "GB_s": round(b / (sort_ms * 1e-3) / 1e9, 1),
                       "frac": round(b / (sort_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    alu = {}
    for k, (f_blend, f_eval) in BLEND_FLOPS.items():
        if stage_ms.get(k, 0) > 0:
            visited = w[1] if k == "blend_bwd" else w[4]
            flops = f_blend * w[0] + f_eval * (visited - w[0])
            ach = flops / (stage_ms[k] * 1e-3) / 1e12
            alu[k] = {"GFLOP": round(flops / 1e9, 3), "ms": round(stage_ms[k], 4), "TFLOP_s": round(ach, 3),
                      "frac": round(ach / FP32_VECTOR_PEAK_TFLOPS, 4),
                      "frac_unpacked": round(ach / FP32_UNPACKED_PEAK_TFLOPS, 4)}

    out = {"it_s": round(it_s, 3), "ms_per_step": round(1e3 * elapsed / args.steps, 4),
           "mpix_per_s": round(cfg.width * cfg.height * it_s / 1e6, 2),
           "step_ms": {"mean": round(float(step_times.mean()), 4), "median": round(float(np.median(step_times)), 4),
                       "min": round(float(step_times.min()), 4), "max": round(float(step_times.max()), 4)},
           "stage_ms": {k: round(v, 4) for k, v in stage_ms.items()}, "stages": group_stages(stage_ms),
           "visible_avg": int(vis_avg), "pairs_avg": int(pairs_avg), "work_per_image": work_avg,
           "blended_per_pixel": round(w[0] / (cfg.width * cfg.height), 2),
           "hbm_stages": hbm, "alu_stages": alu}

    if render:
        # forward only (preprocess, binning, blend): the paper's rendering rate;
        # no backward follows, so the preprocess writes no colour Jacobian for it
        jac = fr.pre.color_jac
        fr.pre.color_jac = None
        for i in range(args.warmup):
            fr.forward(cstructs[i % ncam], st, stream=stream, sync_pairs=False)
        torch.cuda.synchronize()
        t_start = time.perf_counter()
        for i in range(args.steps):
            fr.forward(cstructs[i % ncam], st, stream=stream, sync_pairs=False)
        torch.cuda.synchronize()
        t_r = (time.perf_counter() - t_start) / args.steps
        fr.pre.color_jac = jac
        out["render_only"] = {"it_s": round(1.0 / t_r, 3), "ms_per_frame": round(1e3 * t_r, 4),
                              "mpix_per_s": round(cfg.width * cfg.height / t_r / 1e6, 2)}

    if train:
        # training step: each step followed by the fused Adam update of every
        # parameter tensor (the paper's optimisation comparison)
        from paper_2609_05255_amd.optim import FusedAdam, camera_spacing
        opt = FusedAdam(st, fr, kid, camera_dbar=camera_spacing(np.array([c.campos for c in cams])))
        for i in range(args.warmup):
            step(i)
            opt.step(stream)
        torch.cuda.synchronize()
        t_start = time.perf_counter()
        for i in range(args.steps):
            step(i)
            opt.step(stream)
        torch.cuda.synchronize()
        t_train = (time.perf_counter() - t_start) / args.steps
        timer.attach()
        timer.reset()
        for i in range(args.steps):
            opt.step(stream)
        torch.cuda.synchronize()
        adam_ms, adam_n = timer.read()["adam"]
        gs.Timer.detach()
        adam_ms /= max(adam_n, 1)
        adam_bytes = opt.bytes_per_step()
        adam_gbs = adam_bytes / (adam_ms * 1e-3) / 1e9
        hbm["adam"] = {"algorithmic_MB": round(adam_bytes / 1e6, 1), "ms": round(adam_ms, 4),
                       "GB_s": round(adam_gbs, 1), "frac": round(adam_gbs / HBM_PEAK_GBS, 4)}
        out["train_step"] = {"it_s": round(1.0 / t_train, 3), "ms_per_step": round(1e3 * t_train, 4),
                             "adam_ms": round(adam_ms, 4),
                             "optimizer": "fused Adam over every parameter tensor, one launch per step"}
        if kid == gs.GS_APP_SH3:
            # the same training step with the Adam update applied inside the
            # backward (gs_render_bwd_adam): no gradient is written or read back;
            # that backward reads the coefficients for the update anyway, so its
            # forward writes no colour Jacobian
            jac = fr.pre.color_jac
            fr.pre.color_jac = None

            def train_in_bwd(i):
                c = cstructs[i % ncam]
                fr.forward(c, st, stream=stream, sync_pairs=False)
                opt.backward_step(fr, c, st, grads_up[i % ncam], stream=stream)
            for i in range(args.warmup):
                train_in_bwd(i)
            torch.cuda.synchronize()
            t_start = time.perf_counter()
            for i in range(args.steps):
                train_in_bwd(i)
            torch.cuda.synchronize()
            t_in = (time.perf_counter() - t_start) / args.steps
            timer.attach()
            timer.reset()
            for i in range(args.steps):
                opt.backward_step(fr, cstructs[i % ncam], st, grads_up[i % ncam], stream=stream)
            torch.cuda.synchronize()
            kt_in = timer.read()
            gs.Timer.detach()
            fr.pre.color_jac = jac
            pb_ms, pb_n = kt_in["preprocess_bwd"]
            pb_ms /= max(pb_n, 1)
            out["train_step_adam_in_bwd"] = {
                "it_s": round(1.0 / t_in, 3), "ms_per_step": round(1e3 * t_in, 4),
                "preprocess_bwd_adam_ms": round(pb_ms, 4),
                "optimizer": "the Adam update of the Gaussians' parameters applied inside the preprocess backward"}
        del opt
    timer.close()
    out["_kernel_counts"] = {k: cnt for k, (ms, cnt) in kt.items() if cnt}
    out["_ctx"] = dict(scene=scene, cams=cams, cfg=cfg, frame=fr, st=st, cstructs=cstructs, kid=kid,
                       capacity=capacity, steps_cams=steps_cams, vis_avg=vis_avg)
    return out


def release(m):
    """Frees a measured workload's device buffers."""
    import torch
    m.pop("_ctx", None)
    m.pop("_kernel_counts", None)
    gc.collect()
    torch.cuda.empty_cache()


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the rasterizer runs on a single MI355X "
              "(the multi-GPU data-parallel design is described, not built); use --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2609_05255_amd import gsraster as gs
    from paper_2609_05255_amd import inputs

    torch.cuda.set_device(0)
    cfg = inputs.CONFIGS[args.config]
    kind = args.appearance or cfg.appearance[0]
    arch = None if args.neural_arch is None else tuple(int(v) for v in args.neural_arch.split(","))
    main_m = measure(gs, inputs, torch, args.config, kind, args, arch)
    ctx = main_m["_ctx"]
    stage_ms = main_m["stage_ms"]
    kcount = main_m["_kernel_counts"]

    # roofline of the dominant kernel (largest total time per step)
    dominant = max(stage_ms, key=lambda k: stage_ms[k] * kcount.get(k, 1))
    roofline = None
    if dominant in main_m["hbm_stages"]:
        h = main_m["hbm_stages"][dominant]
        roofline = {"kernel": dominant, "bound": "hbm", "achieved": h["GB_s"], "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": h["frac"], "traffic": None}
    elif dominant in main_m["alu_stages"]:
        a = main_m["alu_stages"][dominant]
        roofline = {"kernel": dominant, "bound": "alu", "achieved": a["TFLOP_s"], "peak": FP32_VECTOR_PEAK_TFLOPS,
                    "unit": "TFLOP/s", "frac": a["frac"], "traffic": None,
                    "peak_unpacked": FP32_UNPACKED_PEAK_TFLOPS, "frac_unpacked": a["frac_unpacked"],
                    "work": "%s GFLOP per launch from gs_render_work's counts: blended entries x %d, other entries "
                            "the method visits x %d" % (a["GFLOP"], *BLEND_FLOPS[dominant])}
    if roofline is not None and dominant in KERNEL_SOURCES:
        tb = recorded_traffic(dominant, ctx["cfg"].name, kind)
        roofline["traffic"] = None if tb is None else round(tb)
        roofline["traffic_unit"] = "bytes per launch"
        roofline["source_hash"] = source_hash(dominant)

    # render only: the unfolded neural decoder against its folded form
    folded = None
    if kind == "neural" and arch in (None, (2, 16, 0)):
        st, fr = ctx["st"], ctx["frame"]
        stream = torch.cuda.current_stream()
        fr_fold = gs.Frame(ctx["scene"].n, ctx["cfg"].width, ctx["cfg"].height, gs.GS_APP_NEURAL_FOLDED,
                           ctx["capacity"])
        timer = gs.Timer()
        timer.attach()
        st.fold_neural(stream)
        torch.cuda.synchronize()
        folded = {"fold_ms": round(timer.read()["neural_fold"][0], 4)}
        for name, frame in (("neural", fr), ("neural_folded", fr_fold)):
            timer.reset()
            for i in range(args.steps):
                frame.forward(ctx["cstructs"][i % len(ctx["cstructs"])], st, stream=stream, sync_pairs=False)
            torch.cuda.synchronize()
            pre_ms, pre_n = timer.read()["preprocess"]
            pre_ms /= max(pre_n, 1)
            gbs = algorithmic_bytes("preprocess", ctx["scene"].n, ctx["vis_avg"], name) / (pre_ms * 1e-3) / 1e9
            folded[name] = {"preprocess_ms": round(pre_ms, 4), "preprocess_GB_s": round(gbs, 1)}
        gs.Timer.detach()
        timer.close()
        del fr_fold

    scene, cams = ctx["scene"], ctx["cams"]
    release(main_m)
    extra = {}
    if not args.no_extra and args.config == "paper_sh3" and kind == "sh3":
        lat = measure(gs, inputs, torch, "paper_latent", "latent", args)
        release(lat)
        extra["latent_vs_sh3"] = {
            "workload": "3M Gaussians, 1600x1064, same geometry and cameras; SH3 (192 B) vs latent + MLP (28 B)",
            "sh3_it_s": main_m["it_s"], "latent_it_s": lat["it_s"], "ratio": round(lat["it_s"] / main_m["it_s"], 4),
            "sh3_train_it_s": main_m["train_step"]["it_s"], "latent_train_it_s": lat["train_step"]["it_s"],
            "train_ratio": round(lat["train_step"]["it_s"] / main_m["train_step"]["it_s"], 4),
            "sh3_train_adam_in_bwd_it_s": main_m.get("train_step_adam_in_bwd", {}).get("it_s"),
            "sh3_render_mpix_s": main_m["render_only"]["mpix_per_s"],
            "latent_render_mpix_s": lat["render_only"]["mpix_per_s"]}
        extra["paper_latent"] = lat
        stress = {}
        for sk in ("sh3", "latent"):
            m = measure(gs, inputs, torch, "stress", sk, args, train=False)
            release(m)
            stress[sk] = m
        extra["stress"] = {"workload": "6M Gaussians, 1920x1080, log-scale N(-5.5, 0.7), 16 cameras", **stress}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(scene, cams, kind)

    out = {
        "metric": METRIC,
        "value": main_m["it_s"],
        "unit": "it/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": main_m["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if kind in ("sh3", "nasg", "nasgabor") else "f32+f16",
        "data": "synthetic",
        "config": {"workload": "%s: %d Gaussians, %dx%d, %s appearance, %d cameras" % (
            ctx["cfg"].name, scene.n, ctx["cfg"].width, ctx["cfg"].height, kind, len(cams)),
            "gaussians": scene.n, "width": ctx["cfg"].width, "height": ctx["cfg"].height, "appearance": kind,
            "cameras": len(cams), **({"neural_arch": list(arch)} if arch else {})},
        "mpix_per_s": main_m["mpix_per_s"],
        "roofline": roofline,
        "cpu_baseline": cpu,
        **{k: v for k, v in main_m.items() if k not in ("it_s", "ms_per_step", "mpix_per_s")},
        **({"neural_folded": folded} if folded else {}),
        **extra,
    }
    print(json.dumps(out), flush=True)


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(scene, cams, kind):
    """The oracle on the host cores, camera 0 of the workload: one full
    iteration (preprocess of every Gaussian, binning, forward and backward
    blending of every tile), measured on all the cores the process may use
    and on one thread."""
    from oracle import oracle as orc
    from paper_2609_05255_amd import inputs

    cam = cams[0]
    g = inputs.make_upstream_grad(cam.width, cam.height, 0)
    tx, ty = orc.tile_grid(cam)
    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    threads = min(cores, int(os.environ.get("OMP_NUM_THREADS", cores)))
    runs = {}
    for label, k in (("all", threads), ("one", 1)):
        orc.set_threads(k)
        print("# cpu baseline: full oracle iteration on %d thread(s)" % k, file=sys.stderr, flush=True)
        t0 = time.perf_counter()
        pre = orc.preprocess(cam, scene, kind=kind)
        t1 = time.perf_counter()
        values, _, ranges = orc.bin_sort(cam, pre)
        t2 = time.perf_counter()
        orc.render_fwd(cam, pre, ranges, values)
        t3 = time.perf_counter()
        orc.render_bwd(cam, scene, pre, ranges, values, g, kind=kind)
        t4 = time.perf_counter()
        del pre, values, ranges
        runs[label] = (t4 - t0, "preprocess %.1f, binning %.1f, forward %.1f, backward %.1f" % (
            t1 - t0, t2 - t1, t3 - t2, t4 - t3))
        print("# cpu baseline: %.1fs" % (t4 - t0), file=sys.stderr, flush=True)
    orc.set_threads(threads)
    what = ("camera 0, one full iteration: preprocess of all %d Gaussians, binning, forward and backward "
            "blending of all %d tiles" % (scene.n, tx * ty))
    return {"value": round(1.0 / runs["all"][0], 6), "unit": "it/s", "cores": threads, "kind": "oracle",
            "sample": "%s, on %d threads: %.1fs (%s)" % (what, threads, runs["all"][0], runs["all"][1]),
            "s_per_iter": round(runs["all"][0], 2), "nproc": os.cpu_count(), "cpu_model": cpu_model(),
            "single_thread": {"value": round(1.0 / runs["one"][0], 6), "unit": "it/s", "cores": 1,
                              "s_per_iter": round(runs["one"][0], 2),
                              "sample": "%s, on one thread: %.1fs (%s)" % (what, runs["one"][0], runs["one"][1])}}


if __name__ == "__main__":
    main()
