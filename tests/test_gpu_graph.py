"""One BOM step captured in a HIP graph (torch's graph capture over the library's launches, which the
binding enqueues on the capture stream) and replayed. The library records no memset, allocation or
synchronisation, so a step captures whole. Every replay is checked against the same step run eagerly on a
twin of the problem, with that eager work and a device synchronisation between the replays: the state
(theta, v, q) and the step's outputs must be bitwise equal after each replay. A replay repeats the
captured step counter t (its bias corrections are kernel arguments), so the eager twin runs the same t."""
import numpy as np
import pytest
import torch

from gpu_util import log, needs_gpu
from synth.workloads import BY_NAME

pytestmark = [pytest.mark.gpu, needs_gpu]


def _bits(t):
    a = t.detach().cpu()
    return a.view(torch.int16).numpy() if a.dtype == torch.bfloat16 else a.numpy().view(np.uint8)


@pytest.mark.parametrize("name", ["tiny_linear_c10", "vision_head_c1000", "lm_small_v32000"])
def test_step_graph_replays_match_eager(name):
    import bench

    w = BY_NAME[name]
    dev = torch.device("cuda:0")
    log(f"[graph] {name}: two twins, eager warmup")
    pg, pe = bench.Problem(w, dev), bench.Problem(w, dev)
    pg.step(1)
    pe.step(1)
    torch.cuda.synchronize()
    t = 2
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        pg.step(t)
    torch.cuda.synchronize()
    for r in range(3):
        g.replay()
        pe.step(t)                      # eager work between the replays
        torch.cuda.synchronize()
        for k in ("theta", "v", "q", "q_hat", "u", "dH"):
            assert np.array_equal(_bits(getattr(pg, k)), _bits(getattr(pe, k))), f"replay {r}: {k}"
        for k in ("s", "row_lse", "row_argmax", "loss", "n_valid", "flags"):
            assert np.array_equal(_bits(pg.res[k]), _bits(pe.res[k])), f"replay {r}: {k}"
        assert np.array_equal(_bits(pg.R), _bits(pe.R)), f"replay {r}: R"
        log(f"    replay {r}: bitwise equal to the eager step")
    del g, pg, pe
    torch.cuda.empty_cache()
