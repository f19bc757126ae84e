"""Split-row residual with the partner exchange switched off from the host.

When rows are too wide for one workgroup, several workgroups share each row and exchange their
per-part (max, sum, argmax) records; every wait is bounded and, past the bound, a workgroup reduces
the missing part's slice from Z itself with the operations that part runs, in the same order. A poll
limit below zero (environment BOM_RESIDUAL_SPIN, read once per process) takes that path for every part
of every row, so this test runs the library in a child process with it set, checks the results against
the oracle like any other parity case, and checks that every output is bitwise equal to the normal
path's (run in this process); the flags word differs only by BOM_FLAG_RESIDUAL_RECOMPUTED.
"""
import os
import subprocess
import sys
import tempfile

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import gen_labels, gen_matrix, log, needs_gpu
from paper_2609_36738_amd import bom
from test_gpu_parity import _compare_residual

pytestmark = [pytest.mark.gpu, needs_gpu]

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
# the multirow cases give each row group several rows (a workgroup prefetches the next row during one)
CASES = [("split3_v70000_multirow", 300, 70000), ("split4_v100008", 24, 100008),
         ("split4_v128256_multirow", 200, 128256), ("split10_v300000", 8, 300000), ("split16_v520000", 6, 520000),
         ("split16_v520000_multirow", 40, 520000)]

CHILD = r"""
import sys
import numpy as np
import torch
sys.path.insert(0, {root!r})
sys.path.insert(0, {tests!r})
import synth
from gpu_util import gen_labels, gen_matrix
from paper_2609_36738_amd import bom
N, V, out_path = {N}, {V}, {out!r}
print(f"[child] split fallback N={{N}} V={{V}}", flush=True)
_, Zd = gen_matrix(N, V, synth.STREAM_Z, 1.28, "bf16")
y = gen_labels(N, V, "zipf", 0.05, 2)
o = bom.bom_residual(Zd, torch.from_numpy(y).to("cuda:0"))
torch.cuda.synchronize()
np.savez(out_path, **{{k: (o[k].float() if k == "R" else o[k]).cpu().numpy()
                      for k in ("s", "row_lse", "row_argmax", "row_target", "R", "loss", "n_valid", "flags")}})
print("[child] done", flush=True)
"""


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_split_rows_without_exchange(case):
    name, N, V = case
    log(f"[residual] {name}: child process with BOM_RESIDUAL_SPIN=-1")
    with tempfile.TemporaryDirectory() as td:
        out = os.path.join(td, "out.npz")
        code = CHILD.format(root=ROOT, tests=os.path.join(ROOT, "tests"), N=N, V=V, out=out)
        env = dict(os.environ, BOM_RESIDUAL_SPIN="-1")
        r = subprocess.run([sys.executable, "-u", "-c", code], env=env, cwd=ROOT, timeout=240,
                           capture_output=True, text=True)
        log(r.stdout[-2000:])
        assert r.returncode == 0, r.stderr[-4000:]
        got = np.load(out)
        # npz arrays as torch tensors, like the binding's outputs, for the shared comparison
        res = {k: torch.from_numpy(np.asarray(got[k])) for k in got.files}
    Zh, Zd = gen_matrix(N, V, synth.STREAM_Z, 1.28, "bf16")
    y = gen_labels(N, V, "zipf", 0.05, 2)
    orc = oracle.residual(Zh, y)
    flags_fb = int(res["flags"][0])
    assert flags_fb & bom.BOM_FLAG_RESIDUAL_RECOMPUTED, "the fallback path must report the recomputation"
    res["flags"] = res["flags"] & ~bom.BOM_FLAG_RESIDUAL_RECOMPUTED
    _compare_residual(name, Zh, y, res, orc, "bf16")
    # the normal path (exchange on) in this process: the same bits everywhere
    log(f"[residual] {name}: normal path, bitwise comparison")
    ref = bom.bom_residual(Zd, torch.from_numpy(y).to("cuda:0"))
    torch.cuda.synchronize()
    assert int(ref["flags"][0]) == flags_fb & ~bom.BOM_FLAG_RESIDUAL_RECOMPUTED
    for k in ("s", "row_lse", "row_argmax", "row_target", "loss", "n_valid"):
        a, b = ref[k].cpu().numpy(), res[k].numpy()
        assert a.dtype == b.dtype and np.array_equal(a.view(np.uint32), b.view(np.uint32)), k
    assert np.array_equal(ref["R"].float().cpu().numpy().view(np.uint32), res["R"].numpy().view(np.uint32)), "R"
