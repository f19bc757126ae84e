"""The allocation-free residual (bom_residual_noalloc): the library's fixed device scratch array in
place of the caller's workspace. Checked through the C-ABI against bom_residual with its own workspace
on the same inputs, on two calls in a row, the second with a smaller input (a narrower vocabulary on the
LDS-parked rows after a split-row call that also uses the exchange records): the scratch keeps the first
call's contents, so the second must not depend on them. The kernels and launch shapes are the same, so
the outputs are bitwise equal. A shape beyond the scratch is refused before anything is enqueued."""
import numpy as np
import pytest
import torch

import synth
from gpu_util import gen_labels, gen_matrix, log, needs_gpu
from paper_2609_36738_amd import bom

pytestmark = [pytest.mark.gpu, needs_gpu]

KEYS = ("s", "row_lse", "row_argmax", "row_target", "R", "loss", "n_valid", "flags")


def _outputs(N, V, dev):
    return dict(s=torch.empty(V, device=dev), row_lse=torch.empty(N, device=dev),
                row_argmax=torch.empty(N, dtype=torch.int32, device=dev), row_target=torch.empty(N, device=dev),
                R=torch.empty((N, V), dtype=torch.bfloat16, device=dev), loss=torch.empty(1, device=dev),
                n_valid=torch.empty(1, dtype=torch.int32, device=dev), flags=torch.empty(1, dtype=torch.int32, device=dev))


def _bits(t):
    a = t.cpu()
    if a.dtype == torch.bfloat16:
        a = a.view(torch.int16)
    return a.numpy().view(np.uint8)


def test_noalloc_matches_workspace_entry_two_calls():
    dev = torch.device("cuda:0")
    # first: split rows (two workgroups per row, exchange records in the scratch); second: smaller
    for N, V, std in [(2048, 60000, 1.28), (1000, 32000, 0.55)]:
        log(f"[noalloc] N={N} V={V}")
        need = bom.load().bom_residual_workspace_bytes(N, V, bom.BOM_BF16)
        assert need <= bom.RESIDUAL_SCRATCH_BYTES
        _, Zd = gen_matrix(N, V, synth.STREAM_Z, std, "bf16")
        yd = torch.from_numpy(gen_labels(N, V, "zipf", 0.05, 2)).to(dev)
        out = _outputs(N, V, dev)
        bom.bom_residual_noalloc(Zd, yd, **out)
        ref = bom.bom_residual(Zd, yd)
        torch.cuda.synchronize()
        for k in KEYS:
            assert np.array_equal(_bits(out[k]), _bits(ref[k])), k
        assert int(out["n_valid"][0]) > 0


def test_noalloc_refuses_a_shape_beyond_the_scratch():
    dev = torch.device("cuda:0")
    N, V = 512, 70000
    need = bom.load().bom_residual_workspace_bytes(N, V, bom.BOM_BF16)
    assert need > bom.RESIDUAL_SCRATCH_BYTES
    Zd = torch.zeros((N, V), dtype=torch.bfloat16, device=dev)
    yd = torch.zeros(N, dtype=torch.int32, device=dev)
    out = _outputs(N, V, dev)
    with pytest.raises(bom.BomError) as ei:
        bom.bom_residual_noalloc(Zd, yd, **out)
    assert ei.value.status == 5 and "scratch" in ei.value.detail
