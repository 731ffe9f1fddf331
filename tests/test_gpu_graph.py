"""The allocation-free step under HIP stream capture: one step of a mixed
stack captured into a graph and replayed several times, with eager work and
synchronizations between the replays; every replay must equal, bit for bit,
the same step run eagerly on a copy of the same buffers.  The captured step
keeps its arguments (the same t, hence the same orientation and sketch), and
reads whatever the buffers hold at replay time.
"""
import sys

import pytest

torch = pytest.importorskip("torch")

from paper_2609_36692_amd import normpre as N  # noqa: E402
from paper_2609_36692_amd import workloads as WL  # noqa: E402

pytestmark = pytest.mark.gpu

# Plain and Gram-space Newton-Schulz items, wide and tall, a ragged one.
SHAPES = [(256, 256), (200, 450), (450, 200), (130, 70)]


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("variant", ["G", "L"])
def test_captured_noalloc_step_replays_match_eager(variant):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    dev = torch.device("cuda:0")
    ctx = N.normpre_init(0)
    try:
        mats = []
        for i, shape in enumerate(SHAPES):
            wl = WL.Workload("g", 70 + i, [shape], "lowrank", 1.0, rank=8)
            mats.append(WL.make_matrix(wl, 0, "cpu", shape=shape))
        graph_bufs = [[m[j].to(dev).clone() for m in mats] for j in range(3)]
        eager_bufs = [[x.clone() for x in bufs] for bufs in graph_bufs]
        hp = N.normpre_default_hparams(lr=1e-2, weight_decay=0.1, step=1, rank=8)
        v = N.VARIANTS[variant]
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            # One eager step on each set first (both now hold the same state,
            # and the context's last stream is the capture stream).
            N.normpre_step_noalloc(ctx, v, *graph_bufs, hp)
            N.normpre_step_noalloc(ctx, v, *eager_bufs, hp)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            N.normpre_step_noalloc(ctx, v, *graph_bufs, hp)
        torch.cuda.synchronize()
        for r in range(3):
            _say(f"{variant} replay {r}")
            g.replay()
            torch.cuda.synchronize()
            with torch.cuda.stream(s):
                N.normpre_step_noalloc(ctx, v, *eager_bufs, hp)
            torch.cuda.synchronize()
            for j, name in ((0, "W"), (2, "M")):
                for a, b in zip(graph_bufs[j], eager_bufs[j]):
                    assert torch.isfinite(a).all()
                    assert torch.equal(a, b), (variant, r, name)
            # Eager work between replays: new gradients in both sets.
            for a, b in zip(graph_bufs[1], eager_bufs[1]):
                a.mul_(-0.5).add_(0.01)
                b.copy_(a)
            torch.cuda.synchronize()
        del g
    finally:
        N.normpre_destroy(ctx)
