"""The layer forward captured into a HIP graph (through torch.cuda.graph) and
replayed: every replay must give the eager result's bits.  Replays alternate
with eager work and synchronisations, and the captured sequence includes a
budget upload and the shared expert's side stream (fork and join by events),
as the decode benchmark's captured steps do.
"""
import numpy as np
import pytest

from paper_2606_27866_amd import flexmoe as fm
from paper_2606_27866_amd import synth
from tests.gpu_util import mini_layer, say

CASES = [
    # name, T, d, E, I, k, I_s  (T <= 64: decode kernels; larger: prefill tiles)
    ("g_decode", 8, 256, 16, 192, 4, 128),
    ("g_decode1", 1, 256, 16, 192, 4, 128),
    ("g_prefill", 300, 256, 8, 320, 2, 256),
]


@pytest.mark.gpu
@pytest.mark.parametrize("spec", CASES, ids=[c[0] for c in CASES])
def test_gpu_graph_replay_matches_eager(spec):
    import torch
    name, T, d, E, I, k, I_s = spec
    cfg, x, lg, w, s = mini_layer(name, T, d, E, I, k, I_s, config_id=210 + CASES.index(spec))
    layer = fm.Layer(d, E, I, k, I_s, synth.BF16, 0, max_tokens=T)
    layer.set_weights(*[fm.to_device(a) for a in (*w, *s)])
    tables = [np.full(E, I, np.int32), synth.tiny_keep_table(E, I, 5)]
    xd, ld = fm.to_device(x), fm.to_device(lg)
    y = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
    say(name, "eager")
    eager = []
    for t in tables:
        layer.set_budget(t)
        layer.forward(xd, ld, y=y)
        torch.cuda.synchronize()
        eager.append(fm.to_host(y).copy())
    graphs = []
    for t in tables:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            layer.set_budget(t)
            layer.forward(xd, ld, y=y)
        graphs.append(g)
    torch.cuda.synchronize()
    say(name, "replays")
    for rep in range(3):
        for gi, g in enumerate(graphs):
            y.zero_()
            g.replay()
            torch.cuda.synchronize()
            np.testing.assert_array_equal(fm.to_host(y), eager[gi])
            # eager work in between: the other table, outside the graph
            layer.set_budget(tables[1 - gi])
            layer.forward(xd, ld, y=y)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(fm.to_host(y), eager[1 - gi])
