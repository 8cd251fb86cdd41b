"""Benchmark of the rasterizer's forward + backward on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config paper_sh3|paper_latent|stress|medium|tiny]
                    [--no-cpu-baseline]

One step = one full pass of the hot path for one camera of the scene:
gs_preprocess (with the read-back of the pair count), gs_bin_sort, gs_render_fwd
and gs_render_bwd, cycling over the configuration's cameras. Scene parameters
and upstream gradients are resident on the GPU before timing starts. Prints one
JSON line: fwd+bwd iterations/s (and Mpix/s), per-kernel times measured with HIP
events on the rendering stream, the roofline of the dominant kernel, and the
CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "fwd+bwd iterations/sec and rendered Mpix/s at 3M Gaussians, 1600x1064"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
FP32_VECTOR_PEAK_TFLOPS = 157.3
# fp32 work per blended (pixel, splat) pair, counting an FMA as 2 (see the kernels):
# forward: quadratic form 11, exp 2, alpha 2, transmittance 2, weight 1, colour 6;
# backward: quadratic form 11, exp 2, alpha 2, transmittance 2, dcolour 4, dalpha 15,
# suffix sum 6, dopacity + dmean2d + dconic 20.
BLEND_FLOPS_PER_PAIR = {"blend_fwd": 24.0, "blend_bwd": 62.0}


# HBM traffic of a kernel, from memory-counter runs summarised under profiles/
# (FETCH_SIZE and WRITE_SIZE per dispatch, each scaled by what the counter reads
# for a copy of known size). Each summary records a hash of the kernel's
# sources; once they change, the recorded figure no longer describes the
# kernel and the traffic is reported as null.
TRAFFIC_SUMMARIES = {("blend_bwd", "paper_sh3", "sh3"): "profiles/blend_bwd_paper_sh3_traffic.txt"}
KERNEL_SOURCES = {"blend_bwd": ("paper_2609_05255_amd/csrc/blend.hip", "paper_2609_05255_amd/csrc/gs_internal.h")}


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
    ap.add_argument("--cpu-tiles", type=int, default=96, help="tiles in the CPU-baseline sample")
    ap.add_argument("--copy-probe-mb", type=int, default=0,
                    help="before the steps, one device-to-device copy of this many MB (a plain copy kernel of "
                         "known size, to calibrate memory-traffic counters)")
    return ap.parse_args()


def algorithmic_bytes(kernel: str, n: int, vis: float, kind: str, sh_degree: int = 3) -> float | None:
    """HBM bytes a launch must move at minimum (per launch, averaged over cameras)."""
    # appearance bytes per visible Gaussian: SH3 48 fp32, latent 14 binary16, neural a 12 B
    # base colour and 8 binary16 features
    # (the folded form: the base colour and 16 binary16 pre-activations, 44 B; NASG 12 + 32 B,
    # NASGabor 12 + 36 B; 16 raw binary16 features: 12 + 32 B)
    app = (4 * 3 * (sh_degree + 1) ** 2 if kind == "sh3" else
           {"neural_folded": 44, "neural_raw16": 44, "nasg": 44, "nasgabor": 48}.get(kind, 28))
    if kernel == "preprocess":
        # params 44 B + tiles 4 B + depth key 4 B per Gaussian; appearance + 48 B of projected splat
        # (mean 8, conic 12, opacity 4, colour 12, rectangle 8, depth 4) per visible one; the record
        # written is 64 B, the rest being the blend's early-skip fields
        return n * (44 + 8) + vis * (app + 48)
    if kernel == "preprocess_bwd":
        # tiles 4 B + dense gradient writes per Gaussian; params, accumulators and appearance per visible one
        grad = 44 + 4 * {"sh3": 48, "latent": 14, "neural": 11, "neural_raw16": 19, "nasg": 11, "nasgabor": 12}[kind]
        return n * (4 + grad) + vis * (44 + 36 + app)
    return None


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the rasterizer runs on a single MI355X "
              "(the multi-GPU data-parallel design is described, not built); use --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2609_05255_amd import gsraster as gs
    from paper_2609_05255_amd import inputs

    cfg = inputs.CONFIGS[args.config]
    kind = args.appearance or cfg.appearance[0]
    kid = {"sh3": gs.GS_APP_SH3, "latent": gs.GS_APP_LATENT_MLP, "neural": gs.GS_APP_NEURAL,
           "nasg": gs.GS_APP_NASG, "nasgabor": gs.GS_APP_NASGABOR}[kind]
    torch.cuda.set_device(0)
    dev = "cuda:0"
    t0 = time.time()
    arch = None if args.neural_arch is None else tuple(int(v) for v in args.neural_arch.split(","))
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

    # size the pair buffers: preprocess every camera once (untimed)
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

    def step(i):
        c = cstructs[i % len(cstructs)]
        fr.forward(c, st, stream=stream)
        fr.backward(c, st, grads_up[i % len(cstructs)], stream=stream)

    print("# capacity %d pairs; warmup" % capacity, file=sys.stderr, flush=True)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    # timed region
    t_start = time.perf_counter()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    it_s = args.steps / elapsed

    # per-step spread: the same K steps again, a pair of events around each
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for i in range(args.steps):
        ev[i][0].record(stream)
        step(i)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    step_times = np.array([a.elapsed_time(b) for a, b in ev])
    step_spread = {"mean": round(float(step_times.mean()), 4), "median": round(float(np.median(step_times)), 4),
                   "min": round(float(step_times.min()), 4), "max": round(float(step_times.max()), 4)}

    # blended pairs per image (sum of n_contrib), for the blend's work figure
    contrib = []
    for i in range(len(cstructs)):
        fr.forward(cstructs[i], st, stream=stream)
        contrib.append(float(fr.n_contrib.double().sum().item()))
    # per-kernel durations: the same K steps again with HIP events around every kernel
    gs.timing_enable(True)
    gs.timing_reset()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    kt = gs.timing_read()
    gs.timing_enable(False)
    stage_ms = {k: (ms / cnt if cnt else 0.0) for k, (ms, cnt) in kt.items() if cnt}

    # roofline of the dominant kernel
    ncam = len(cstructs)
    steps_cams = [i % ncam for i in range(args.steps)]
    vis_avg = float(np.mean([visible[i] for i in steps_cams]))
    pairs_avg = float(np.mean([pairs[i] for i in steps_cams]))
    dominant = max(stage_ms, key=lambda k: stage_ms[k] * kt[k][1])
    roofline = None
    bkind = "neural_raw16" if kind == "neural" and arch and arch[2] else kind
    hbm_kernels = {k: algorithmic_bytes(k, scene.n, vis_avg, bkind) for k in ("preprocess", "preprocess_bwd")}
    if dominant in hbm_kernels:
        b = hbm_kernels[dominant]
        ach = b / (stage_ms[dominant] * 1e-3) / 1e9
        roofline = {"kernel": dominant, "bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": None}
    else:
        # blend kernels: fp32 vector work per blended (pixel, splat) pair
        flops_per_pair = BLEND_FLOPS_PER_PAIR.get(dominant, None)
        if flops_per_pair is not None:
            e = float(np.mean([contrib[i] for i in steps_cams]))
            ach = e * flops_per_pair / (stage_ms[dominant] * 1e-3) / 1e12
            roofline = {"kernel": dominant, "bound": "alu", "achieved": round(ach, 3),
                        "peak": FP32_VECTOR_PEAK_TFLOPS, "unit": "TFLOP/s",
                        "frac": round(ach / FP32_VECTOR_PEAK_TFLOPS, 4), "traffic": None}
    if roofline is not None and dominant in KERNEL_SOURCES:
        tb = recorded_traffic(dominant, cfg.name, kind)
        roofline["traffic"] = None if tb is None else round(tb)
        roofline["traffic_unit"] = "bytes per launch"
        roofline["source_hash"] = source_hash(dominant)
    hbm_all = {}
    for k, b in hbm_kernels.items():
        if k in stage_ms and stage_ms[k] > 0:
            ach = b / (stage_ms[k] * 1e-3) / 1e9
            hbm_all[k] = {"algorithmic_MB": round(b / 1e6, 1), "ms": round(stage_ms[k], 4),
                          "GB_s": round(ach, 1), "frac": round(ach / HBM_PEAK_GBS, 4)}

    # training step: the same K steps followed each by the fused Adam update of
    # every parameter tensor (the paper's optimisation comparison); value
    # above stays the forward+backward metric
    from paper_2609_05255_amd.optim import FusedAdam, camera_spacing
    opt = FusedAdam(st, fr, kid, camera_dbar=camera_spacing([c.campos for c in cams]))
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
    gs.timing_enable(True)
    gs.timing_reset()
    for i in range(args.steps):
        opt.step(stream)
    torch.cuda.synchronize()
    adam_ms, adam_n = gs.timing_read()["adam"]
    gs.timing_enable(False)
    adam_ms /= max(adam_n, 1)
    adam_bytes = opt.bytes_per_step()
    adam_gbs = adam_bytes / (adam_ms * 1e-3) / 1e9
    hbm_all["adam"] = {"algorithmic_MB": round(adam_bytes / 1e6, 1), "ms": round(adam_ms, 4),
                       "GB_s": round(adam_gbs, 1), "frac": round(adam_gbs / HBM_PEAK_GBS, 4)}
    train = {"it_s": round(1.0 / t_train, 3), "ms_per_step": round(1e3 * t_train, 4), "adam_ms": round(adam_ms, 4),
             "optimizer": "fused Adam over every parameter tensor, one launch per step"}

    # render only (preprocess, binning, forward blend), the unfolded neural
    # decoder against its folded form (the paper's viewer optimisation)
    render_only = None
    if kind == "neural" and arch in (None, (2, 16, 0)):
        fr_fold = gs.Frame(scene.n, cfg.width, cfg.height, gs.GS_APP_NEURAL_FOLDED, capacity, device=dev)
        gs.timing_enable(True)
        gs.timing_reset()
        st.fold_neural(stream)
        torch.cuda.synchronize()
        fold_ms = gs.timing_read()["neural_fold"][0]
        gs.timing_enable(False)
        render_only = {"fold_ms": round(fold_ms, 4)}
        for name, frame in (("neural", fr), ("neural_folded", fr_fold)):
            for i in range(args.warmup):
                frame.forward(cstructs[i % ncam], st, stream=stream)
            torch.cuda.synchronize()
            t_start = time.perf_counter()
            for i in range(args.steps):
                frame.forward(cstructs[i % ncam], st, stream=stream)
            torch.cuda.synchronize()
            t_r = (time.perf_counter() - t_start) / args.steps
            gs.timing_enable(True)
            gs.timing_reset()
            for i in range(args.steps):
                frame.forward(cstructs[i % ncam], st, stream=stream)
            torch.cuda.synchronize()
            pre_ms, pre_n = gs.timing_read()["preprocess"]
            gs.timing_enable(False)
            pre_ms /= max(pre_n, 1)
            gbs = algorithmic_bytes("preprocess", scene.n, vis_avg, name) / (pre_ms * 1e-3) / 1e9
            render_only[name] = {"it_s": round(1.0 / t_r, 3), "ms_per_step": round(1e3 * t_r, 4),
                                 "preprocess_ms": round(pre_ms, 4), "preprocess_GB_s": round(gbs, 1)}
        del fr_fold

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(scene, cams, kind, args.cpu_tiles)

    mpix = cfg.width * cfg.height * it_s / 1e6
    out = {
        "metric": METRIC,
        "value": round(it_s, 3),
        "unit": "it/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(1e3 * elapsed / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if kind in ("sh3", "nasg", "nasgabor") else "f32+f16",
        "data": "synthetic",
        "config": {"workload": "%s: %d Gaussians, %dx%d, %s appearance, %d cameras" % (
            cfg.name, scene.n, cfg.width, cfg.height, kind, ncam),
            "gaussians": scene.n, "width": cfg.width, "height": cfg.height, "appearance": kind,
            "cameras": ncam, **({"neural_arch": list(arch)} if arch else {})},
        "mpix_per_s": round(mpix, 2),
        "visible_avg": int(vis_avg),
        "pairs_avg": int(pairs_avg),
        "blended_pairs_avg": int(np.mean(contrib)),
        "stage_ms": {k: round(v, 4) for k, v in stage_ms.items()},
        "step_ms": step_spread,
        "hbm_stages": hbm_all,
        "roofline": roofline,
        "train_step": train,
        "render_only": render_only,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def cpu_baseline(scene, cams, kind, n_tiles_sample):
    """The oracle on the host: full preprocess of every Gaussian, then binning,
    forward and backward blending restricted to a random sample of tiles, the
    per-tile part scaled to the whole image. One camera, single thread."""
    from oracle import oracle as orc

    cam = cams[0]
    tx, ty = orc.tile_grid(cam)
    T = tx * ty
    rng = np.random.default_rng(0)
    sample = np.sort(rng.choice(T, size=min(n_tiles_sample, T), replace=False))
    print("# cpu baseline: oracle preprocess of %d Gaussians" % scene.n, file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    pre = orc.preprocess(cam, scene, kind=kind)
    t_pre = time.perf_counter() - t0
    print("# cpu baseline: preprocess %.1fs; sampled tiles next" % t_pre, file=sys.stderr, flush=True)
    # keep only Gaussians whose rectangle meets a sampled tile
    sx, sy = sample % tx, sample // tx
    r = pre["rect"]
    keep = np.zeros(scene.n, bool)
    vis = np.nonzero(pre["tiles"] > 0)[0]
    for lo in range(0, vis.size, 1 << 20):
        idx = vis[lo:lo + (1 << 20)]
        hit = ((r[0, idx, None] <= sx[None]) & (sx[None] < r[2, idx, None]) &
               (r[1, idx, None] <= sy[None]) & (sy[None] < r[3, idx, None])).any(axis=1)
        keep[idx[hit]] = True
    sub = orc.Preprocessed({k: v.copy() for k, v in pre.items()})
    sub["tiles"][~keep] = 0
    sub["flags"][~keep] = 0
    t1 = time.perf_counter()
    values, _, ranges = orc.bin_sort(cam, sub)
    mask = np.zeros(T, bool)
    mask[sample] = True
    ranges[~mask] = 0
    img, fT, nc, _ = orc.render_fwd(cam, sub, ranges, values)
    from paper_2609_05255_amd import inputs
    g = inputs.make_upstream_grad(cam.width, cam.height, 0)
    orc.render_bwd(cam, scene, sub, ranges, values, g, kind=kind)
    t_tiles = time.perf_counter() - t1
    scale = T / sample.size
    t_iter = t_pre + t_tiles * scale
    return {"value": round(1.0 / t_iter, 6), "unit": "it/s", "cores": 1, "kind": "oracle",
            "sample": "camera 0: preprocess of all %d Gaussians (%.1fs) + binning, forward and backward "
                      "blending of %d random tiles of %d (%.1fs), tile part scaled x%.1f" % (
                          scene.n, t_pre, sample.size, T, t_tiles, scale),
            "s_per_iter": round(t_iter, 2)}


if __name__ == "__main__":
    main()
