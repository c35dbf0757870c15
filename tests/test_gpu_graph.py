"""The entry points under HIP graph capture: a step of plan, forward and backward
(RoIAlign with the tile gather, and RoI max pooling) captured once with
torch.cuda.CUDAGraph, then replayed several times with eager work and
synchronizations between the replays.  Every replay must reproduce the eager step:
the forward outputs bit for bit (they do not depend on the plan's list order), the
gradients within the backward tolerance against the oracle.

The library allocates nothing, never synchronizes and clears with fill kernels (no
memset nodes), so its calls can be recorded into a graph.
"""
import numpy as np
import pytest

import oracle
import paper_1906_07155_amd as rex
from paper_1906_07155_amd import workloads as W
from gpu_helpers import check_bwd, from_device, log, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rex.lib()


SHAPES = [(2, 96, 24, 40), (2, 96, 12, 20), (2, 96, 6, 10), (2, 96, 3, 5)]
SC = [0.25, 0.125, 0.0625, 0.03125]


def _inputs(seed, K):
    rng = np.random.default_rng(seed)
    feats_np = [rng.standard_normal(s, dtype=np.float32) for s in SHAPES]
    rois = W.draw_rois(rng, 2, K // 2, (96, 160), (4.0, 200.0))
    g = rng.standard_normal((rois.shape[0], 96, 7, 7), dtype=np.float32)
    return feats_np, rois, g


def _replay_and_check(step, outputs, reset, check):
    """Eager step, capture, then three replays each followed by eager work."""
    s = torch.cuda.current_stream()
    step()
    torch.cuda.synchronize()
    eager = [o.clone() for o in outputs]
    side = torch.cuda.Stream()
    side.wait_stream(s)
    with torch.cuda.stream(side):
        step()                      # warm-up on a side stream before capture
    s.wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for r in range(3):
        reset()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        log("replay %d" % r)
        check(eager, r)
        step()                      # eager work between the replays
        torch.cuda.synchronize()


def test_align_step_in_a_graph():
    feats_np, rois_np, g_np = _inputs(600, 160)
    K = rois_np.shape[0]
    feats = [to_device(f, "f32") for f in feats_np]
    rois = torch.from_numpy(rois_np).cuda()
    gout = torch.from_numpy(g_np).cuda()
    levels = torch.empty(K, dtype=torch.int32, device="cuda")
    ws = torch.empty(rex.workspace_size(feats, SC, K), dtype=torch.uint8, device="cuda")
    out = torch.empty((K, 96, 7, 7), device="cuda")
    grads = [torch.empty(s, device="cuda").contiguous(memory_format=torch.channels_last)
             for s in SHAPES]

    def step():
        rex.plan(feats, SC, rois, 56.0, levels_out=levels, workspace=ws)
        rex.roi_align_fwd(feats, SC, rois, levels, (7, 7), 2, True, out=out, workspace=ws)
        rex.roi_align_bwd(gout, rois, levels, (7, 7), 2, True, grads, SC, zero_init=True,
                          workspace=ws, algorithm="gather")

    def reset():
        out.fill_(-1.0)
        for x in grads:
            x.fill_(9.0)

    lv = oracle.level_map(rois_np, 4, 56.0)
    g64 = g_np.astype(np.float64)
    gref = oracle.roi_align_bwd(g64, SHAPES, SC, rois_np, lv, 7, 7, 2, True, "parity")
    aref = oracle.roi_align_bwd(np.abs(g64), SHAPES, SC, rois_np, lv, 7, 7, 2, True, "parity")

    def check(eager, r):
        assert torch.equal(out, eager[0]), "replay %d: forward differs from the eager step" % r
        for l in range(4):
            check_bwd(from_device(grads[l]), gref[l], aref[l], False,
                      "replay %d gradient level %d" % (r, l))

    _replay_and_check(step, [out], reset, check)


def test_pool_step_in_a_graph():
    feats_np, rois_np, g_np = _inputs(601, 160)
    K = rois_np.shape[0]
    feats = [to_device(f, "f32") for f in feats_np]
    rois = torch.from_numpy(rois_np).cuda()
    gout = torch.from_numpy(g_np).cuda()
    levels = torch.empty(K, dtype=torch.int32, device="cuda")
    ws = torch.empty(rex.workspace_size(feats, SC, K), dtype=torch.uint8, device="cuda")
    out = torch.empty((K, 96, 7, 7), device="cuda")
    am = torch.empty((K, 96, 7, 7), dtype=torch.int32, device="cuda")
    grads = [torch.empty(s, device="cuda").contiguous(memory_format=torch.channels_last)
             for s in SHAPES]

    def step():
        rex.plan(feats, SC, rois, 56.0, levels_out=levels, workspace=ws)
        rex.roi_pool_fwd(feats, SC, rois, levels, (7, 7), out=out, argmax=am, workspace=ws)
        rex.roi_pool_bwd(gout, am, rois, levels, grads, SC, zero_init=True, workspace=ws)

    def reset():
        out.fill_(-1.0)
        am.fill_(-7)
        for x in grads:
            x.fill_(9.0)

    lv = oracle.level_map(rois_np, 4, 56.0)
    f64 = [f.astype(np.float64) for f in feats_np]
    _, am_ref = oracle.roi_pool_fwd(f64, SC, rois_np, lv, 7, 7)
    g64 = g_np.astype(np.float64)
    gref = oracle.roi_pool_bwd(g64, am_ref, SHAPES, rois_np, lv)
    aref = oracle.roi_pool_bwd(np.abs(g64), am_ref, SHAPES, rois_np, lv)

    def check(eager, r):
        assert torch.equal(out, eager[0]) and torch.equal(am, eager[1]), (
            "replay %d: forward differs from the eager step" % r)
        for l in range(4):
            check_bwd(from_device(grads[l]), gref[l], aref[l], False,
                      "replay %d gradient level %d" % (r, l))

    _replay_and_check(step, [out, am], reset, check)
