"""libbom.so without a GPU: it loads, exports every entry point include/bom.h declares, and rejects
bad arguments on the host before any HIP call (fake non-null pointers are never dereferenced)."""
import ctypes
import os
import re

import pytest
import torch

from paper_2609_36738_amd import bom

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = ctypes.c_void_p(0x1000)      # never dereferenced: validation fails first
FAKE2 = ctypes.c_void_p(0x9000000)


def _declared():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            text = open(os.path.join(ROOT, "include", fn)).read()
            names |= set(re.findall(r"^[A-Za-z_][\w \*]*?\b(bom_\w+)\s*\(", text, flags=re.M))
    return names


@pytest.fixture(scope="module")
def lib():
    return bom.load()


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert {"bom_residual", "bom_ema", "bom_head_vjp", "bom_update"} <= names
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings(lib):
    for code in range(9):
        assert lib.bom_status_string(code).decode().startswith("BOM_")
    assert lib.bom_version() >= 100


def _res(lib, **kw):
    a = dict(Z=FAKE, dt=bom.BOM_BF16, N=8, V=16, ldz=16, labels=FAKE, ig=-100, s=FAKE, lse=FAKE, am=None, tg=None,
             R=FAKE2, rdt=bom.BOM_BF16, ldr=16, loss=FAKE, nv=FAKE, fl=FAKE, ws=ctypes.c_void_p(0x100000), wsb=1 << 30)
    a.update(kw)
    return lib.bom_residual(a["Z"], a["dt"], a["N"], a["V"], a["ldz"], a["labels"], a["ig"], a["s"], a["lse"], a["am"],
                            a["tg"], a["R"], a["rdt"], a["ldr"], a["loss"], a["nv"], a["fl"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(Z=None), 1), (dict(labels=None), 1), (dict(s=None), 1), (dict(lse=None), 1), (dict(fl=None), 1),
    (dict(N=0), 2), (dict(V=1), 2), (dict(ldz=15), 2), (dict(ldr=8), 2), (dict(N=1 << 31), 2),
    (dict(dt=7), 3), (dict(rdt=bom.BOM_F32), 3),
    (dict(ws=None), 5), (dict(wsb=16), 5), (dict(ws=ctypes.c_void_p(0x100010)), 5),
    (dict(R=ctypes.c_void_p(0x1010)), 6),
])
def test_residual_rejects(lib, kw, code):
    assert _res(lib, **kw) == code
    assert lib.bom_last_error().decode() != ""


def test_residual_workspace_query(lib):
    assert lib.bom_residual_workspace_bytes(0, 10, 0) == 0
    a = lib.bom_residual_workspace_bytes(4096, 32000, 1)
    assert a >= 256 * 32000 * 4 and a % 256 == 0


@pytest.mark.parametrize("args,code", [
    ((None, FAKE, 10, 0.9, 1, FAKE2), 1), ((FAKE, FAKE, 0, 0.9, 1, FAKE2), 2),
    ((FAKE, FAKE, 10, 1.0, 1, FAKE2), 4), ((FAKE, FAKE, 10, -0.1, 1, FAKE2), 4), ((FAKE, FAKE, 10, 0.9, 0, FAKE2), 4),
    ((FAKE, FAKE, 10, float("nan"), 1, FAKE2), 4), ((FAKE, FAKE, 10, 0.9, 1, ctypes.c_void_p(0x1004)), 6),
])
def test_ema_rejects(lib, args, code):
    assert lib.bom_ema(*args, None) == code


def _vjp(lib, **kw):
    a = dict(H=FAKE, ldh=64, W=FAKE, ldw=100, R=FAKE, isr=1, ldr=100, dt=bom.BOM_BF16, N=32, d=64, V=100, labels=FAKE,
             ig=-100, lse=None, qh=FAKE, s=FAKE, nv=FAKE, lam=0.5, dW=FAKE, dwdt=bom.BOM_F32, lddw=100, beta=0.0, db=None,
             dH=None, dhdt=bom.BOM_BF16, lddh=64, ws=ctypes.c_void_p(0x100000), wsb=1 << 30)
    a.update(kw)
    return lib.bom_head_vjp(a["H"], a["ldh"], a["W"], a["ldw"], a["R"], a["isr"], a["ldr"], a["dt"], a["N"], a["d"],
                            a["V"], a["labels"], a["ig"], a["lse"], a["qh"], a["s"], a["nv"], a["lam"], a["dW"],
                            a["dwdt"], a["lddw"], a["beta"], a["db"], a["dH"], a["dhdt"], a["lddh"], a["ws"], a["wsb"],
                            None)


@pytest.mark.parametrize("kw,code", [
    (dict(H=None), 1), (dict(dW=None), 1), (dict(nv=None), 1), (dict(db=FAKE, s=None), 1),
    (dict(isr=0), 1),                                # the logits input needs row_lse
    (dict(isr=2), 2), (dict(isr=-1), 2),
    (dict(N=0), 2), (dict(V=1), 2), (dict(ldh=63), 2), (dict(lddw=99), 2), (dict(dH=FAKE, lddh=10), 2),
    (dict(dt=5), 3), (dict(dH=FAKE, dhdt=9), 3), (dict(dwdt=4), 3),
    (dict(dwdt=bom.BOM_BF16, wsb=0), 5),           # bf16 dW needs its fp32 staging in the workspace
    (dict(lam=1.5), 4), (dict(lam=-0.1), 4), (dict(beta=float("inf")), 4),
    (dict(ws=None), 5), (dict(wsb=0), 5),
])
def test_head_vjp_rejects(lib, kw, code):
    assert _vjp(lib, **kw) == code


def _upd(lib, P=1000, segs=(), wd=0.0, v_col=None, ws=None, wsb=0, h=None, **cfgkw):
    c = dict(lr=1e-3, beta2=0.999, eps=1e-8, t=1)
    c.update(cfgkw)
    cfg = bom.make_update_cfg(**c)
    arr = (bom.bom_segment * max(1, len(segs)))(*[bom.bom_segment(*s) for s in segs])
    return lib.bom_update(ctypes.c_void_p(0x100000), ctypes.c_void_p(0x200000), v_col, ctypes.c_void_p(0x300000), h, P,
                          arr, len(segs), wd, ctypes.byref(cfg), ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(P=0), 2), (dict(segs=[(0, 2000, 0.1)]), 2), (dict(segs=[(-1, 2, 0.1)]), 2),
    (dict(segs=[(0, 1, float("nan"))]), 4), (dict(beta2=1.0), 4), (dict(t=0), 4), (dict(eps=0.0), 4),
    (dict(lr=float("inf")), 4), (dict(lam=2.0), 4), (dict(wd=float("nan")), 4), (dict(u_scale=float("nan")), 4),
    (dict(v_col=FAKE), 2), (dict(h=ctypes.c_void_p(0x100100)), 6),
    (dict(factored=True), 1), (dict(factored=True, v_col=ctypes.c_void_p(0x400000), block_cols=6), 8),
    (dict(factored=True, v_col=ctypes.c_void_p(0x400000), P=1002), 8),
    (dict(factored=True, v_col=ctypes.c_void_p(0x400000), block_cols=64, block_rows=8), 5),
    (dict(clip_norm=-1.0), 4), (dict(clip_norm=float("inf")), 4),
    (dict(clip_norm=1.0), 5),                        # dense clipping needs its workspace
])
def test_update_rejects(lib, kw, code):
    assert _upd(lib, **kw) == code


TILE = [(0, 600, 0.1), (600, 400, 0.0)]
BIG_WS = dict(ws=ctypes.c_void_p(0x4000000), wsb=1 << 30)


@pytest.mark.parametrize("kw,code", [
    (dict(segs=TILE, blocks=[768, 1], v_col=FAKE, **BIG_WS), 2),          # v_col must be NULL
    (dict(segs=[], blocks=[], **BIG_WS), 1),                              # segments are required
    (dict(segs=[(0, 600, 0.1), (601, 399, 0.0)], blocks=[4, 4], **BIG_WS), 2),   # a gap
    (dict(segs=[(0, 600, 0.1), (600, 300, 0.0)], blocks=[4, 4], **BIG_WS), 2),   # ends before P
    (dict(segs=[(0, 600, 0.1), (600, 0, 0.0), (600, 400, 0.0)], blocks=[4, 4, 4], **BIG_WS), 2),  # empty segment
    (dict(segs=TILE, blocks=[0, 4], **BIG_WS), 2),                        # block length 0
    (dict(segs=TILE, blocks=[4, 4], state_dtype=torch.bfloat16, **BIG_WS), 3),   # fp32 state only
    (dict(segs=TILE, blocks=[4, 4]), 5),                                  # workspace required
    (dict(segs=TILE, blocks=[4, 4], ws=ctypes.c_void_p(0x4000010), wsb=1 << 30), 5),   # 256-byte alignment
])
def test_update_blocks_rejects(lib, kw, code):
    assert _upd(lib, **kw) == code


def test_update_blocks_alias_and_workspace_bound(lib):
    cfg = bom.make_update_cfg(lr=1e-3, beta2=0.999, eps=1e-8, t=1, blocks=[4, 4])
    segs = (bom.bom_segment * 2)(*[bom.bom_segment(*s) for s in TILE])
    # v (250 block entries) overlapping theta
    assert lib.bom_update(ctypes.c_void_p(0x100000), ctypes.c_void_p(0x100100), None, ctypes.c_void_p(0x300000), None,
                          1000, segs, 2, 0.0, ctypes.byref(cfg), ctypes.c_void_p(0x4000000), 1 << 30, None) == 6
    # the partial-sum bound: ceil(n / blk) ceil(blk / 4096) <= 3 n / 4096 + 1 pieces per segment
    for P in (1, 4096, 10**6, 8 * 10**9):
        nb = lib.bom_update_workspace_bytes(P, ctypes.byref(cfg))
        assert nb >= 4 * (3 * P / 4096 + 16) and nb % 256 == 0
    for n, blk in ((4097, 4097), (10**6, 4097), (10**6, 8191), (5000, 10**7), (49152 * 7 + 5, 49152)):
        pieces = -(-n // blk) * -(-min(blk, n) // 4096)
        assert pieces <= 3 * n / 4096 + 1


def test_update_null_pointers(lib):
    cfg = bom.make_update_cfg(lr=1e-3, beta2=0.999, eps=1e-8, t=1)
    assert lib.bom_update(None, FAKE, None, FAKE, None, 10, None, 0, 0.0, ctypes.byref(cfg), None, 0, None) == 1
    assert lib.bom_update(FAKE, FAKE, None, FAKE, None, 10, None, 0, 0.0, None, None, 0, None) == 1
    assert lib.bom_update(FAKE, FAKE, None, FAKE, None, 10, None, 3, 0.0, ctypes.byref(cfg), None, 0, None) == 2


def test_update_workspace_query(lib):
    dense = bom.make_update_cfg(lr=1e-3, beta2=0.999, eps=1e-8, t=1)
    assert lib.bom_update_workspace_bytes(10**6, ctypes.byref(dense)) == 0
    clipped = bom.make_update_cfg(lr=1e-3, beta2=0.999, eps=1e-8, t=1, clip_norm=1.0)
    assert lib.bom_update_workspace_bytes(10**6, ctypes.byref(clipped)) > 0
    fac_c = bom.make_update_cfg(lr=1e-3, beta2=0.999, eps=1e-8, t=1, factored=True, clip_norm=1.0)
    fac_n = bom.make_update_cfg(lr=1e-3, beta2=0.999, eps=1e-8, t=1, factored=True)
    assert lib.bom_update_workspace_bytes(1 << 24, ctypes.byref(fac_c)) > lib.bom_update_workspace_bytes(
        1 << 24, ctypes.byref(fac_n))
    fac = bom.make_update_cfg(lr=1e-3, beta2=0.999, eps=1e-8, t=1, factored=True)
    P = 476 * 4096 * 4096 + 3429 * 4096
    assert lib.bom_update_workspace_bytes(P, ctypes.byref(fac)) > 0


def _tele(lib, **kw):
    a = dict(H=FAKE, ldh=64, hdt=bom.BOM_BF16, R=FAKE, ldr=100, rdt=bom.BOM_BF16, N=32, d=64, V=100, labels=FAKE,
             ig=-100, s=FAKE, qh=FAKE, nv=FAKE, MW=ctypes.c_void_p(0x100000), ldm=100, Mb=None, beta1=0.9, t=1,
             out=ctypes.c_void_p(0x900000), ws=ctypes.c_void_p(0x2000000), wsb=1 << 30)
    a.update(kw)
    return lib.bom_head_telemetry(a["H"], a["ldh"], a["hdt"], a["R"], a["ldr"], a["rdt"], a["N"], a["d"], a["V"],
                                  a["labels"], a["ig"], a["s"], a["qh"], a["nv"], a["MW"], a["ldm"], a["Mb"], a["beta1"],
                                  a["t"], a["out"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(H=None), 1), (dict(MW=None), 1), (dict(out=None), 1), (dict(N=0), 2), (dict(ldm=99), 2),
    (dict(ldr=10), 2), (dict(hdt=7), 3), (dict(beta1=1.0), 4), (dict(t=0), 4), (dict(wsb=0), 5),
    (dict(Mb=ctypes.c_void_p(0x100000 + 400)), 6),
])
def test_head_telemetry_rejects(lib, kw, code):
    assert _tele(lib, **kw) == code


def test_head_forward_rejects(lib):
    assert lib.bom_head_forward(FAKE, 8, FAKE, 4, None, 5, 4, 8, 4, FAKE2, 4, None) == 3
    assert lib.bom_head_forward(FAKE, 7, FAKE, 4, None, bom.BOM_F32, 4, 8, 4, FAKE2, 4, None) == 2
    assert lib.bom_head_forward(None, 8, FAKE, 4, None, bom.BOM_F32, 4, 8, 4, FAKE2, 4, None) == 1


def test_residual_noalloc_refuses_beyond_scratch(lib):
    # the size check runs before the scratch is looked up or anything is enqueued (no GPU needed)
    N, V = 512, 70000
    assert lib.bom_residual_workspace_bytes(N, V, bom.BOM_BF16) > bom.RESIDUAL_SCRATCH_BYTES
    st = lib.bom_residual_noalloc(FAKE, bom.BOM_BF16, N, V, V, FAKE, -100, FAKE, FAKE, None, None, None, bom.BOM_BF16,
                                  V, FAKE, FAKE, FAKE, None)
    assert st == 5 and b"scratch" in lib.bom_last_error()
    assert lib.bom_residual_noalloc(None, bom.BOM_BF16, 8, 100, 100, FAKE, -100, FAKE, FAKE, None, None, None,
                                    bom.BOM_BF16, 100, FAKE, FAKE, FAKE, None) == 1


def _adamw(lib, P=1000, beta1=0.9, v_col=None, ws=None, wsb=0, m=ctypes.c_void_p(0x500000), **cfgkw):
    c = dict(lr=1e-3, beta2=0.999, eps=1e-8, t=1)
    c.update(cfgkw)
    cfg = bom.make_update_cfg(**c)
    arr = (bom.bom_segment * 1)()
    return lib.bom_adamw_update(ctypes.c_void_p(0x100000), m, ctypes.c_void_p(0x200000), v_col,
                                ctypes.c_void_p(0x300000), P, arr, 0, 0.0, beta1, ctypes.byref(cfg), ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(m=None), 1), (dict(P=0), 2), (dict(beta1=1.0), 4), (dict(beta1=-0.5), 4), (dict(t=0), 4),
    (dict(clip_norm=1.0), 8), (dict(state_dtype=__import__("torch").bfloat16), 8),
    (dict(v_col=FAKE), 2), (dict(m=ctypes.c_void_p(0x100100)), 6),
    (dict(factored=True), 1), (dict(factored=True, v_col=ctypes.c_void_p(0x400000), block_cols=512), 8),
    (dict(factored=True, v_col=ctypes.c_void_p(0x400000), block_cols=1024, P=1002), 8),
    (dict(factored=True, v_col=ctypes.c_void_p(0x400000), block_cols=1024, P=4096), 5),
])
def test_adamw_update_rejects(lib, kw, code):
    assert _adamw(lib, **kw) == code
