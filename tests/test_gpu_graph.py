"""A whole training step (gs_preprocess, gs_bin_sort with the pair count on
the device, gs_render_fwd, gs_render_bwd) captured in a HIP graph on the
caller's stream, once per camera, and replayed: the library launches only
kernels in a step (no allocation, no memset, no host synchronisation), so
every replay must give what the eager step gives. Replays are interleaved
with eager steps and synchronisations; the lists, ranges, image, final
transmittance and last contributors must be the same bits, and the gradients
agree to the parity bar (they differ in the float atomics' summation order)."""
import pytest
import torch

from paper_2609_05255_amd import gsraster as gs
from paper_2609_05255_amd import inputs
from parity import say

pytestmark = pytest.mark.gpu

GRADS = ("dmeans", "dlog_scales", "dquats", "dopacity_logits", "dsh", "dlatent", "dmlp_w")


def outputs(fr):
    # the pair buffer past P keeps whatever an earlier step left there
    P = int(fr.num_pairs.item())
    out = {k: getattr(fr, k).clone() for k in ("ranges", "image", "final_T", "n_contrib")}
    out["values"] = fr.values[:P].clone()
    for k in GRADS:
        t = getattr(fr, k, None)
        if t is not None:
            out[k] = t.clone()
    return out


def check_close(a, b, kind, label):
    """Two GPU runs that differ in the float atomics' summation order, held to
    the parity bar: every element within 1e-3 |b| + 1e-5 max|b| and relative
    L2 <= 1e-4 (a sum with heavy cancellation can move by more than 1e-4 of
    itself between orders). Past the decoder a last-bit difference can also
    move a binary16 rounding to the neighbouring value, so there the decoder
    bar applies: at most 0.2% of the elements beyond that bound and none
    beyond 20 times it."""
    d = (a - b).abs()
    m = float(b.abs().max())
    bound = 1e-3 * b.abs() + 1e-5 * m
    rel = float(torch.linalg.vector_norm(a - b) / max(float(torch.linalg.vector_norm(b)), 1e-30))
    assert rel <= 1e-4, (label, rel)
    if kind == "sh3":
        assert bool((d <= bound).all()), (label, float(d.max()))
        return
    assert float((d > bound).float().mean()) <= 2e-3, label
    assert bool((d <= 20 * bound).all()), label


@pytest.mark.parametrize("kind", ["sh3", "latent"])
def test_step_in_a_graph(kind):
    kid = {"sh3": gs.GS_APP_SH3, "latent": gs.GS_APP_LATENT_MLP}[kind]
    sc = inputs.make_scene("medium", appearance=(kind,))
    cams = inputs.make_cameras("medium")[:3]
    say("case graph %s: %d Gaussians, %d cameras" % (kind, sc.n, len(cams)))
    st = gs.SceneTensors(sc)
    cs = [gs.camera_struct(c) for c in cams]
    ups = [torch.from_numpy(inputs.make_upstream_grad(c.width, c.height, i)).cuda() for i, c in enumerate(cams)]
    probe = gs.Frame(sc.n, cams[0].width, cams[0].height, kid, 1)
    g, app = st.gaussians(), st.appearance(kid)
    cap = max(gs.gs_preprocess(c, g, app, probe.pre, probe.workspace, probe.ws_bytes) for c in cs) + 4096
    del probe
    fr = gs.Frame(sc.n, cams[0].width, cams[0].height, kid, cap)
    s = torch.cuda.Stream()

    def step(i):
        fr.forward(cs[i], st, sync_pairs=False)
        fr.backward(cs[i], st, ups[i])

    with torch.cuda.stream(s):
        for i in range(len(cs)):
            step(i)
    torch.cuda.synchronize()
    ref = []
    for i in range(len(cs)):
        with torch.cuda.stream(s):
            step(i)
        torch.cuda.synchronize()
        assert not fr.pairs_overflowed()
        ref.append(outputs(fr))
    graphs = []
    for i in range(len(cs)):
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr, stream=s):
            step(i)
        graphs.append(gr)
    torch.cuda.synchronize()
    for rep in range(3):
        for i in range(len(cs)):
            graphs[i].replay()
            torch.cuda.synchronize()
            got = outputs(fr)
            for k in ("values", "ranges", "image", "final_T", "n_contrib"):
                assert torch.equal(got[k], ref[i][k]), (rep, i, k)
            for k in GRADS:
                if k in got:
                    check_close(got[k], ref[i][k], kind, (rep, i, k))
        # eager work between the replays
        with torch.cuda.stream(s):
            step(rep % len(cs))
        torch.cuda.synchronize()
    say("  %d replays of %d graphs match the eager steps" % (3 * len(cs), len(cs)))
