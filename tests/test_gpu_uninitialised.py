"""No call reads device memory it has not written: before each call torch's allocator cache is filled with NaN,
so the outputs and workspaces the call receives (allocated right after) start as NaN, and any word a kernel
reads before writing it shows up as NaN in the results. Inputs are finite. The cases cover every residual route
(register rows, including a spare chunk per thread; LDS-parked rows; split rows; two passes; scalar and strided
layouts), the head VJP routes (fused small launches, SIMT with k splits, 256-tile whole rounds and leftovers,
the paired launch, the logits route, lambda = 0), the forward and the fused forward + residual, and the update
layouts with clipping, bf16 state, blocks and AdamW."""
import numpy as np
import pytest
import torch

import synth
from gpu_util import gen_labels, gen_matrix, log, needs_gpu
from paper_2609_36738_amd import bom

pytestmark = [pytest.mark.gpu, needs_gpu]


def dev():
    return torch.device("cuda:0")


def poison(gib=2):
    x = torch.empty(int(gib * (1 << 30) // 4), dtype=torch.float32, device=dev())
    x.fill_(float("nan"))
    torch.cuda.synchronize()
    del x   # back to torch's cache, not to the driver: the next allocations reuse it


def no_nan(tag, **ts):
    torch.cuda.synchronize()
    for k, t in ts.items():
        if t is None or not t.is_floating_point():
            continue
        n = int(torch.isnan(t.float()).sum().item())
        assert n == 0, f"{tag}: {n} NaN in {k}"


def _residual(N, V, dt, pad=0, write_R=True):
    _, Zd = gen_matrix(N, V, synth.STREAM_Z, 0.55, dt)
    y = torch.from_numpy(gen_labels(N, V, "zipf" if V > 1000 else "uniform", 0.05)).to(dev())
    poison()
    R = torch.empty((N, V + pad), dtype=Zd.dtype, device=dev())[:, :V] if pad else None
    res = bom.bom_residual(Zd, y, R=R, write_R=write_R)
    no_nan(f"residual {N}x{V} {dt} pad={pad}", s=res["s"], row_lse=res["row_lse"], row_target=res["row_target"],
           loss=res["loss"], R=res["R"] if write_R else None)
    return Zd, y, res


RESIDUAL = [(300, 2050, "bf16", 0), (64, 10000, "f32", 0), (300, 2056, "bf16", 4), (256, 10, "f32", 0),
            (40, 70003, "f32", 0), (8, 330000, "bf16", 0), (600, 50304, "bf16", 0), (200, 128256, "bf16", 0),
            (300, 1000, "bf16", 0), (1000, 3000, "bf16", 8), (513, 5000, "f32", 3)]


@pytest.mark.parametrize("case", RESIDUAL, ids=[f"{c[0]}x{c[1]}_{c[2]}_pad{c[3]}" for c in RESIDUAL])
def test_residual_writes_before_reading(case):
    N, V, dt, pad = case
    log(f"[uninitialised] residual {N}x{V} {dt} pad={pad}")
    _residual(N, V, dt, pad)
    _residual(N, V, dt, pad, write_R=False)


VJP = [(256, 128, 10, "f32", 0.5, False, 0), (600, 300, 700, "f32", 0.5, False, 0),
       (200, 64, 333, "bf16", 0.5, False, 0), (1024, 768, 1000, "bf16", 0.5, False, 0),
       (64, 128, 32000, "bf16", 0.5, False, 0), (2056, 520, 6000, "bf16", 0.5, False, 0),
       (2056, 520, 6000, "bf16", 0.0, False, 0), (24600, 520, 2056, "bf16", 0.5, False, 4),
       (4096, 768, 32000, "bf16", 0.5, False, 0), (4096, 768, 32000, "bf16", 0.5, True, 0),
       (256, 128, 10, "f32", 0.5, True, 0)]


@pytest.mark.parametrize("case", VJP, ids=[f"{c[0]}x{c[1]}x{c[2]}_{c[3]}_lam{c[4]}_z{int(c[5])}_pad{c[6]}" for c in VJP])
def test_head_vjp_writes_before_reading(case):
    N, d, V, dt, lam, zroute, pad = case
    log(f"[uninitialised] head VJP {N}x{d}x{V} {dt} lambda={lam} logits={zroute} pad={pad}")
    _, Hd = gen_matrix(N, d, synth.STREAM_H, 1.0, dt)
    _, Wd = gen_matrix(d, V, synth.STREAM_W, 0.02, dt)
    Zd, y, res = _residual(N, V, dt, pad)
    qh = bom.bom_ema(torch.zeros(V, device=dev()), res["s"], 0.9, 2)
    for dh_dtype in (None, torch.float32):
        poison()
        g = bom.bom_head_vjp(Hd, Wd, Zd if zroute else res["R"], y, qh, res["n_valid"], s=res["s"], lam=lam,
                             want_db=True, dh_dtype=dh_dtype, row_lse=res["row_lse"] if zroute else None)
        no_nan("head VJP", dW=g["dW"], db=g["db"], dH=g["dH"])
    if dt == "bf16" and pad == 0:
        poison()
        no_nan("forward", Z=bom.bom_head_forward(Hd, Wd, None))
        poison()
        fr = bom.bom_head_forward_residual(Hd, Wd, y)
        no_nan("forward + residual", **{k: v for k, v in fr.items() if isinstance(v, torch.Tensor)})


UPDATE = [dict(P=1_000_003), dict(P=1_000_003, off=1), dict(P=1_000_000, clip=0.5), dict(P=1_000_000, bf16=True),
          dict(P=64 * 1024 * 5 + 76, factored=True), dict(P=64 * 1024 * 5 + 76, factored=True, clip=0.5),
          dict(P=1_000_000, blocks=[1, 4096]), dict(P=1_000_000, blocks=[100_000, 50]), dict(P=1_000_003, adamw=True),
          dict(P=64 * 1024 * 5 + 76, factored=True, adamw=True)]


@pytest.mark.parametrize("case", UPDATE, ids=["_".join(f"{k}{v}" for k, v in c.items() if k != "blocks") +
                                              ("_blocks" if "blocks" in c else "") for c in UPDATE])
def test_update_writes_before_reading(case):
    P, off = case["P"], case.get("off", 0)
    factored, clip, bf16 = case.get("factored", False), case.get("clip", 0.0), case.get("bf16", False)
    blocks, adamw = case.get("blocks"), case.get("adamw", False)
    log(f"[uninitialised] update {case}")
    dtp = torch.bfloat16 if bf16 else torch.float32
    g = torch.Generator(device=dev())
    g.manual_seed(7)
    th = (torch.randn(P + off, device=dev(), generator=g) * 0.02).to(dtp)[off:]
    u = (torch.randn(P + off, device=dev(), generator=g) * 1e-3).to(dtp)[off:]
    segs = [(0, P // 2, 0.1), (P // 2, P - P // 2, 0.0)]
    cfg = bom.make_update_cfg(lr=1e-3, beta2=0.999, eps=1e-8, t=2, factored=factored, block_rows=64, block_cols=1024,
                              clip_norm=clip, clip_stats=torch.zeros(2, device=dev()) if clip else None,
                              state_dtype=dtp, blocks=blocks)
    vc = None
    if factored:
        nrows = (P + 1023) // 1024
        v = torch.zeros(nrows, device=dev())
        vc = torch.zeros(((nrows + 63) // 64) * 1024, device=dev())
    elif blocks is not None:
        v = torch.zeros(bom.blocks_count(segs, blocks), device=dev())
    else:
        v = torch.zeros(P + off, device=dev()).to(dtp)[off:]
    poison()
    if adamw:
        m = torch.zeros(P, device=dev())
        bom.bom_adamw_update(th, m, v, u, cfg, v_col=vc, segments=segs)
        no_nan("AdamW", theta=th, m=m, v=v, v_col=vc)
    else:
        bom.bom_update(th, v, u, cfg, v_col=vc, segments=segs)
        no_nan("update", theta=th, v=v, v_col=vc)
