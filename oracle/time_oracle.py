"""Times the CPU oracle on the host: one iteration per camera (preprocess,
binning, forward and backward blending of every tile), single-threaded and on
every core the process may use. Test and measurement infrastructure.

    python oracle/time_oracle.py [--configs tiny,medium,paper_sh3,paper_latent]
                                 [--cameras tiny=1,medium=8,paper_sh3=2,paper_latent=2]
                                 [--single-cameras paper_sh3=1,paper_latent=1] [--out FILE]

Prints one JSON object: the host (CPU model, nproc, threads used) and, per
configuration and thread count, the seconds of each camera's iteration and
their mean, with the Mpix/s that follows.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))

from oracle import oracle as orc  # noqa: E402
from paper_2609_05255_amd import inputs  # noqa: E402


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def one_iteration(cam, scene, kind) -> dict:
    g = inputs.make_upstream_grad(cam.width, cam.height, 0)
    t0 = time.perf_counter()
    pre = orc.preprocess(cam, scene, kind=kind)
    t1 = time.perf_counter()
    values, _, ranges = orc.bin_sort(cam, pre)
    t2 = time.perf_counter()
    orc.render_fwd(cam, pre, ranges, values)
    t3 = time.perf_counter()
    orc.render_bwd(cam, scene, pre, ranges, values, g, kind=kind)
    t4 = time.perf_counter()
    return {"s": t4 - t0, "preprocess": t1 - t0, "bin_sort": t2 - t1, "fwd": t3 - t2, "bwd": t4 - t3}


def parse_counts(text: str) -> dict:
    out = {}
    for item in filter(None, text.split(",")):
        k, v = item.split("=")
        out[k] = int(v)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--configs", default="tiny,medium,paper_sh3,paper_latent")
    ap.add_argument("--cameras", default="tiny=1,medium=8,paper_sh3=2,paper_latent=2",
                    help="cameras timed on all cores")
    ap.add_argument("--single-cameras", default="tiny=1,medium=8,paper_sh3=1,paper_latent=1",
                    help="cameras timed on one thread")
    ap.add_argument("--out", default=None)
    args = ap.parse_args()
    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    threads_all = min(cores, int(os.environ.get("OMP_NUM_THREADS", cores)))
    ncam_all, ncam_one = parse_counts(args.cameras), parse_counts(args.single_cameras)
    res = {"cpu_model": cpu_model(), "nproc": os.cpu_count(), "threads_all": threads_all, "configs": {}}
    for name in filter(None, args.configs.split(",")):
        cfg = inputs.CONFIGS[name]
        kind = cfg.appearance[0]
        scene = inputs.make_scene(cfg, appearance=(kind,))
        cams = inputs.make_cameras(cfg)
        entry = {"gaussians": cfg.n, "width": cfg.width, "height": cfg.height, "appearance": kind}
        for label, threads, count in (("one_thread", 1, ncam_one.get(name, 1)),
                                      ("all_cores", threads_all, ncam_all.get(name, 1))):
            orc.set_threads(threads)
            runs = []
            for i in range(min(count, len(cams))):
                r = one_iteration(cams[i], scene, kind)
                runs.append(r)
                print("# %s %s camera %d: %.2fs" % (name, label, i, r["s"]), file=sys.stderr, flush=True)
            mean = sum(r["s"] for r in runs) / len(runs)
            entry[label] = {"threads": threads, "cameras": len(runs), "s_per_iter": round(mean, 3),
                            "it_s": round(1.0 / mean, 5),
                            "mpix_per_s": round(cfg.width * cfg.height / mean / 1e6, 4),
                            "per_camera_s": [round(r["s"], 3) for r in runs],
                            "stages_s": {k: round(sum(r[k] for r in runs) / len(runs), 3)
                                         for k in ("preprocess", "bin_sort", "fwd", "bwd")}}
        res["configs"][name] = entry
    text = json.dumps(res)
    if args.out:
        with open(args.out, "w") as f:
            f.write(text + "\n")
    print(text, flush=True)


if __name__ == "__main__":
    main()
