"""Head-VJP kernel routes selected by environment variables (read once per process), each run in a
child process and checked against the oracle like the default-path parity cases.

* BOM_VJP_WAVES = "4,4,4,4": the 256 x 256 tiles of dH, dW, the paired launch and the forward on four
  waves per workgroup (one per SIMD, each 128 x 128) instead of eight: whole rounds with leftover split-k
  tiles for dW and for dH, ragged tiles in m, n and k, the paired launch of both products, the forward.
* BOM_VJP_XCD_BLOCK = "0": the plain XCD tile order (2 outer tiles x all 16 inner tiles per XCD round) at
  d = 4096, where the default is the blocked order.
* BOM_VJP_PLAN = "4,3,4,2": the 256-tile rank-1 kernel with k split three ways (dW) and two ways (dH) on
  every tile, followed by the split-k reduction with the rank-1 term.
* BOM_VJP_PLAN = "1,0,1,0": the 128-tile kernels that fold the history into G while staging R (no
  fused small-product launch), with their own k splits.
"""
import os
import subprocess
import sys
import tempfile

import numpy as np
import pytest

import oracle
from gpu_util import log, needs_gpu, rel_fro
from test_gpu_parity import B1, LAM, _vjp_inputs, f32

pytestmark = [pytest.mark.gpu, needs_gpu]

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# name, N, d, V, sampled dW columns, sampled dH rows (None: all)
CASES = [
    ("dW_leftover", 1032, 520, 24000, np.r_[0:40, 21700:21830, 23950:24000], np.r_[0:8, 1024:1032]),
    ("dH_leftover", 24600, 520, 2056, np.r_[0:16, 2040:2056], np.r_[0:32, 21740:21790, 24570:24600]),
    ("tile256_ragged_mnk", 2056, 520, 6000, None, None),
    ("pair_lm_small", 4096, 768, 32000, np.r_[0:64, 31900:32000], np.r_[0:32, 4064:4096]),
]

CHILD = r"""
import sys
import numpy as np
import torch
sys.path.insert(0, {root!r})
sys.path.insert(0, {tests!r})
from paper_2609_36738_amd import bom
from test_gpu_parity import B1, LAM, _vjp_inputs
N, d, V, out_path = {N}, {d}, {V}, {out!r}
print(f"[child] N={{N}} d={{d}} V={{V}}", flush=True)
Hh, Hd, Wh, Wd, Zh, Zd, y, q_prev, t = _vjp_inputs(N, d, V, "bf16", 0.05)
yd = torch.from_numpy(y).to("cuda:0")
res = bom.bom_residual(Zd, yd)
q = torch.from_numpy(q_prev.copy()).to("cuda:0")
qh = bom.bom_ema(q, res["s"], B1, t)
g = bom.bom_head_vjp(Hd, Wd, res["R"], yd, qh, res["n_valid"], s=res["s"], lam=LAM, want_db=True,
                     dh_dtype=torch.float32)
Z = bom.bom_head_forward(Hd, Wd, None)
torch.cuda.synchronize()
np.savez(out_path, dW=g["dW"].double().cpu().numpy(), dH=g["dH"].double().cpu().numpy(),
         Z=Z[:64].double().cpu().numpy())
print("[child] done", flush=True)
"""


VARIANTS = [("BOM_VJP_WAVES", "4,4,4,4", c) for c in CASES] + [
    ("BOM_VJP_PLAN", "4,3,4,2", CASES[0]),
    ("BOM_VJP_PLAN", "4,3,4,2", CASES[2]),
    ("BOM_VJP_PLAN", "1,0,1,0", CASES[2]),
    ("BOM_VJP_PLAN", "1,0,1,0", ("short_128", 640, 256, 3000, None, None)),
    ("BOM_VJP_XCD_BLOCK", "0", ("d4096_plain_order", 10248, 4096, 12000, np.r_[0:64, 11940:12000],
                                np.r_[0:16, 10230:10248])),
]


@pytest.mark.parametrize("var", VARIANTS, ids=[f"{v[0]}={v[1]}-{v[2][0]}" for v in VARIANTS])
def test_env_variant(var):
    env_name, env_value, case = var
    name, N, d, V, cols, rows = case
    log(f"[env variant] {name}: child process with {env_name}={env_value}")
    with tempfile.TemporaryDirectory() as td:
        out = os.path.join(td, "out.npz")
        code = CHILD.format(root=ROOT, tests=os.path.join(ROOT, "tests"), N=N, d=d, V=V, out=out)
        env = dict(os.environ, **{env_name: env_value})
        r = subprocess.run([sys.executable, "-u", "-c", code], env=env, cwd=ROOT, timeout=240,
                           capture_output=True, text=True)
        log(r.stdout[-2000:])
        assert r.returncode == 0, r.stderr[-4000:]
        got = np.load(out)
        Hh, _, Wh, _, Zh, _, y, q_prev, t = _vjp_inputs(N, d, V, "bf16", 0.05)
    o = oracle.residual(Zh, y, want_R=False)
    _, qho = oracle.ema(q_prev, o["s"], f32(B1), t)
    cols = np.arange(V) if cols is None else cols
    rows = np.arange(N) if rows is None else rows
    dW = oracle.dW_cols(Hh, Zh, y, o["row_lse"], qho, o["n_valid"], LAM, cols=cols)
    dH = oracle.dH_rows(Wh, Zh, y, o["row_lse"], qho, o["n_valid"], LAM, rows=rows)
    e_dw, e_dh = rel_fro(got["dW"][:, cols], dW), rel_fro(got["dH"][rows], dH)
    Zo = oracle.head_forward(Hh[:64], Wh, None)
    e_z = rel_fro(got["Z"], Zo)
    log(f"    rel err dW={e_dw:.3e} dH={e_dh:.3e} Z={e_z:.3e}")
    assert e_dw <= 2e-2 and e_dh <= 2e-2 and e_z <= 2e-2
    assert np.isfinite(got["dW"]).all() and np.isfinite(got["dH"]).all()
