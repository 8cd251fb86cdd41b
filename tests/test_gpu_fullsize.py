"""Parity at the full workload sizes, in the benchmark's launch configuration.

The oracle cannot render a 1600x1064 image of 3M Gaussians in a test's time,
so each case checks:
  * the preprocess of every Gaussian, bit-exact against the oracle's;
  * the whole sorted pair list through properties that admit exactly one list
    (given the per-Gaussian tile counts and rectangles checked before);
  * the per-tile lists, image, final transmittance and last contributor on a
    sample of tiles (random ones, the densest one and ragged edge tiles),
    against the oracle rendering only the Gaussians that reach those tiles;
  * properties of every pixel: final transmittance at least the stop
    threshold, last contributor inside its tile's list, no negative colour;
  * every Gaussian's gradient, for an upstream gradient that is zero outside
    the sampled tiles (and on their pixels flagged by the decision margin):
    the oracle's backward over those tiles alone is then the whole backward,
    and every Gaussian that reaches none of them must get an exact zero.
"""
import numpy as np
import pytest

from paper_2609_05255_amd import inputs
from oracle import oracle as orc
from parity import (IMG_ATOL, IMG_RTOL, MARGIN, MLP_GRADS, MLP_HALF_ATOL, NEURAL_FLIP, check_grads,
                    check_list_properties, compare_preprocess, flagged_pixels, grad_stats, lobe_color_atol,
                    report_grads, run_gpu, say, tile_of_ranges)

pytestmark = pytest.mark.gpu

N_RANDOM_TILES = 24
T_STOP = float(np.float32(1e-4))      # the stop threshold as the fp32 kernels hold it


def list_lengths(pre, tiles_x, tiles_y):
    """Pairs per tile from the tile rectangles (2-D difference array)."""
    vis = pre["tiles"] > 0
    r = pre["rect"][:, vis].astype(np.int64)
    d = np.zeros((tiles_y + 1, tiles_x + 1), np.int64)
    np.add.at(d, (r[1], r[0]), 1)
    np.add.at(d, (r[1], r[2]), -1)
    np.add.at(d, (r[3], r[0]), -1)
    np.add.at(d, (r[3], r[2]), 1)
    return d.cumsum(0).cumsum(1)[:tiles_y, :tiles_x].ravel()


def sample_tiles(lengths, tiles_x, tiles_y, seed):
    rng = np.random.default_rng(seed)
    pick = set(rng.choice(tiles_x * tiles_y, size=N_RANDOM_TILES, replace=False).tolist())
    pick.add(int(np.argmax(lengths)))                  # the longest list
    pick.add(tiles_x * tiles_y - 1)                    # bottom-right corner
    pick.add((tiles_y - 1) * tiles_x + tiles_x // 2)   # bottom row (ragged when H % 16 != 0)
    return np.array(sorted(pick), np.int64)


def restrict(pre, sample, tiles_x):
    """The preprocess result with every Gaussian that reaches no sampled tile
    marked culled; returns it and the mask of the Gaussians kept."""
    sx, sy = sample % tiles_x, sample // tiles_x
    r = pre["rect"]
    keep = np.zeros(pre["tiles"].size, bool)
    vis = np.nonzero(pre["tiles"] > 0)[0]
    for lo in range(0, vis.size, 1 << 18):
        idx = vis[lo:lo + (1 << 18)]
        hit = ((r[0, idx, None] <= sx[None]) & (sx[None] < r[2, idx, None]) &
               (r[1, idx, None] <= sy[None]) & (sy[None] < r[3, idx, None])).any(axis=1)
        keep[idx[hit]] = True
    sub = orc.Preprocessed({k: v.copy() for k, v in pre.items()})
    sub["tiles"][~keep] = 0
    sub["flags"][~keep] = 0
    return sub, keep


def tile_pixels(sample, tiles_x, W, H):
    m = np.zeros((H, W), bool)
    for t in sample:
        x0, y0 = (t % tiles_x) * 16, (t // tiles_x) * 16
        m[y0:y0 + 16, x0:x0 + 16] = True
    return m


@pytest.mark.parametrize("config,kind,cam_index,arch", [("paper_sh3", "sh3", 3, None),
                                                         ("paper_latent", "latent", 9, None),
                                                         ("paper_neural", "neural", 7, None),
                                                         ("paper_neural", "neural", 5, (2, 32, 0)),
                                                         ("paper_nasg", "nasg", 11, None),
                                                         ("paper_nasgabor", "nasgabor", 13, None),
                                                         ("stress", "sh3", 5, None),
                                                         ("stress", "latent", 10, None),
                                                         ("stress", "neural", 2, None)])
def test_full_size_sampled(config, kind, cam_index, arch):
    latent = kind in ("latent", "neural")
    sc = inputs.make_scene(config, appearance=(kind,), neural_arch=arch)
    cam = inputs.make_cameras(config)[cam_index]
    W, H = cam.width, cam.height
    tiles_x, tiles_y = orc.tile_grid(cam)
    say("case full-size %s %s%s camera %d: n=%d %dx%d" % (config, kind, "" if arch is None else " %d-%d-%d" % arch,
                                                          cam_index, sc.n, W, H))

    pre = orc.preprocess(cam, sc, kind=kind, half_act=latent)
    P_ref = int(pre["tiles"].astype(np.int64).sum())
    lengths = list_lengths(pre, tiles_x, tiles_y)
    assert lengths.sum() == P_ref
    sample = sample_tiles(lengths, tiles_x, tiles_y, seed=cam_index)
    in_sample = tile_pixels(sample, tiles_x, W, H)
    # the oracle on the sampled tiles first: its decision margins decide which
    # pixels get an upstream gradient
    sub, keep = restrict(pre, sample, tiles_x)
    values, _, ranges = orc.bin_sort(cam, sub)
    unsampled = np.ones(tiles_x * tiles_y, bool)
    unsampled[sample] = False
    ranges_s = ranges.copy()
    ranges_s[unsampled] = 0
    img, fT, n_contrib, margin = orc.render_fwd(cam, sub, ranges_s, values)
    flagged = flagged_pixels(margin, label="sampled ", region=in_sample)
    dL = (inputs.make_upstream_grad(W, H, cam_index) * (in_sample & ~flagged)[None]).astype(np.float32)
    say("  P=%d, %d sampled tiles (longest list %d)" % (P_ref, sample.size, lengths.max()))

    gpu = run_gpu(sc, cam, kind, 3, dL, capacity=P_ref + 4096, extras=False)
    say("  GPU done")

    # preprocess of every Gaussian and the whole list
    flip = NEURAL_FLIP if kind == "neural" else None
    atol = (MLP_HALF_ATOL if latent else
            lobe_color_atol(sc, cam, kind, pre["color"]) if kind in ("nasg", "nasgabor") else 2e-6)
    compare_preprocess(gpu, pre, color_atol=atol, flip=flip)
    assert gpu["P"] == P_ref
    key = np.where(pre["tiles"] > 0, pre["depth"].astype(np.float32).view(np.uint32), np.uint32(0xFFFFFFFF))
    tile_of = tile_of_ranges(gpu["ranges"], gpu["P"])
    check_list_properties(gpu["values"], tile_of, pre["tiles"], pre["rect"], key, tiles_x)
    assert np.array_equal(gpu["ranges"][:, 1] - gpu["ranges"][:, 0], lengths)
    say("  preprocess and list OK")

    # every pixel: properties that hold at any size
    nc = gpu["n_contrib"].astype(np.int64)
    tile_len = lengths.reshape(tiles_y, tiles_x).repeat(16, 0).repeat(16, 1)[:H, :W]
    assert np.all(nc <= tile_len)
    assert np.all(gpu["final_T"] >= T_STOP) and np.all(gpu["final_T"] <= 1.0)
    assert np.all(gpu["image"] >= 0.0)

    # sampled tiles against the oracle
    for t in sample:
        a, b = gpu["ranges"][t]
        c, d = ranges[t]
        assert np.array_equal(gpu["values"][a:b].astype(np.int64), values[c:d].astype(np.int64)), t
    ok = in_sample & (margin > MARGIN)
    atol, rtol = ((flip[0] if flip else MLP_HALF_ATOL), 0.0) if latent else (IMG_ATOL, IMG_RTOL)
    err = np.abs(gpu["image"] - img)
    bad = (err > atol + rtol * np.abs(img)) & ok[None]
    assert not bad.any(), (int(bad.sum()), float(err[:, ok].max()))
    assert np.array_equal(gpu["n_contrib"][ok], n_contrib[ok])
    assert np.all(np.abs(gpu["final_T"] - fT)[ok] <= IMG_ATOL + IMG_RTOL * np.abs(fT[ok]))
    say("  image on %d sampled pixels OK (%d within the decision margin)" % (int(in_sample.sum()),
                                                                             int((in_sample & ~ok).sum())))

    # gradients of every Gaussian
    ref = orc.render_bwd(cam, sc, sub, ranges_s, values, dL, kind=kind, half_act=latent)
    names = ["dmeans", "dlog_scales", "dquats", "dopacity_logits"] + {
        "sh3": ["dsh"], "latent": ["dlatent", "dmlp_w"], "neural": ["dbase_color", "dfeatures", "dmlp_w"],
        "nasg": ["dbase_color", "dlobes"], "nasgabor": ["dbase_color", "dlobes"]}[kind]
    st = grad_stats(gpu["grads"], ref, names)
    report_grads(st)
    if latent:
        check_grads(st, **MLP_GRADS)
    else:
        check_grads(st)
    for k in names:
        if k != "dmlp_w":
            assert np.all(gpu["grads"][k][..., ~keep] == 0), k
    say("  %d Gaussians reach the sample; the other %d have zero gradients" % (int(keep.sum()),
                                                                             int((~keep).sum())))
