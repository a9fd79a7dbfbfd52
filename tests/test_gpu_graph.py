"""The benchmarked step replayed from a captured graph against the same step run eagerly.

Two layer states are set up from the same inputs.  One runs the step (loops 2..R) eagerly, the other
captures it once in a graph and replays it; after every step both states must agree bit for bit (the
kernels are deterministic), with eager work and synchronizations between the replays.  Workloads: the
32K workload's structure at a small size (a band: loop 2 as the subtract pass, the commit and the add
pass), one without a band (the same loop 2 form on the segment kernels without a band), and one whose
column list is above the segment kernels' 2048 entries (loop 2 in the two-pass kernel with its separate
commit and copy refresh)."""
import os
import sys

import numpy as np
import pytest
import torch

from gpu_util import down, down_bits16, say, up_bf16
from workloads import get, make_layer

pytestmark = pytest.mark.gpu

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))


def _state(gs):
    return ([down(t) for t in (gs.o, gs.lse, gs.cand, gs.term, gs.mass, gs.slot_prev)]
            + [down_bits16(t) for t in (gs.k_hat, gs.v_hat, gs.v16)])


@pytest.mark.parametrize("name,over", [("C4", dict(seq=2000, heads=2, window=128, col_budget=4 + 128 + 300)),
                                       ("C2", dict(seq=1500, heads=2, col_budget=200)),
                                       ("C2", dict(seq=2600, heads=2, col_budget=2100))])
def test_graph_replay_matches_eager_steps(F, name, over):
    import bench
    from paper_2609_29812_amd import driver
    w = get(name).replace(**over)
    st = make_layer(w)
    dev = {n: [up_bf16(a) for a in getattr(st, n)] for n in "qkv"}
    say(f"graph replay {w.name} N={w.seq} H={w.heads} window={w.window} list={w.col_budget}")
    states = [driver.setup(dev["q"][0], dev["k"][0], dev["v"][0], w.base_bits, w.group, w.n_sink, w.top_cols,
                           w.window) for _ in range(2)]
    eager = bench.Step(w, dev, states[0], F, torch)
    replay = bench.Step(w, dev, states[1], F, torch)
    graph = bench.capture_step(replay, torch)
    assert graph is not None, "capture failed"
    for step in range(4):
        eager.run()
        graph.replay()
        torch.cuda.synchronize()
        a, b = _state(states[0]), _state(states[1])
        for i, (x, y) in enumerate(zip(a, b)):
            assert np.array_equal(x, y), f"step {step}: state field {i} differs between replay and eager"
        # eager work of the program's own between replays
        scratch = torch.empty(1 << 20, device="cuda").normal_()
        float(scratch.sum())
    say(f"  {step + 1} replays bit-identical to the eager steps")
