"""GPU parity at the full workload sizes, in the launch configurations the benchmark times.

Residual: every row's statistics and the batch-mean residual s are checked in full (the oracle runs
on row chunks in fp64 and the chunk means are combined by their valid-row counts); residual rows on
a sample. Head VJP: 256 sampled dW columns (among them one in each leftover tile band and the ragged
last column) and 256 dH rows (every 256-row tile); the oracle takes only those slices of Z, plus the
dW row-sum invariant over the whole matrix. Update: sampled chunks (dense) or blocks (factored)
whose inputs come from the seeded generator; the rest of the flat buffer holds other seeded values
and is checked by a property (|step| <= lr at t = 1). Forward: sampled rows against the oracle, and the fused
forward + residual against the forward and bom_residual on the same logits.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import bf16_tensor, dev, log, needs_gpu, rel_fro, to_f64
from synth.workloads import BY_NAME
from paper_2609_36738_amd import bom

pytestmark = [pytest.mark.gpu, needs_gpu]

LM = ["lm_small_v32000", "lm_1b_v50304", "lm_8b_v128256"]
f32 = lambda x: float(np.float32(x))


@pytest.fixture(scope="module", params=LM)
def lm(request):
    w = BY_NAME[request.param]
    N, d, V = w.N, w.d, w.V
    log(f"[full] {w.name}: generating inputs")
    zb = synth.normal_bf16(N * V, synth.STREAM_Z, w.logit_std)
    y = synth.labels_zipf(N, V)
    Zd = bf16_tensor(zb, (N, V))
    Zh = synth.bf16_to_f32(zb).reshape(N, V)
    del zb
    yd = torch.from_numpy(y).to(dev())
    log(f"[full] {w.name}: GPU residual")
    res = bom.bom_residual(Zd, yd)
    torch.cuda.synchronize()
    g = {k: res[k].cpu().numpy() for k in ("s", "row_lse", "row_argmax", "row_target", "loss", "n_valid", "flags")}
    rows_R = np.unique(np.r_[np.linspace(0, N - 1, 24).astype(int), [N - 1]])
    g["R_rows"] = to_f64(res["R"][torch.from_numpy(rows_R).to(dev())])
    log(f"[full] {w.name}: oracle residual on row chunks")
    chunk = max(64, (1 << 25) // V)
    lse = np.zeros(N)
    am = np.zeros(N, np.int32)
    tg = np.zeros(N)
    s_num = np.zeros(V)
    ce_num = 0.0
    nv = 0
    flags = 0
    for r0 in range(0, N, chunk):
        o = oracle.residual(Zh[r0:r0 + chunk], y[r0:r0 + chunk], want_R=False)
        lse[r0:r0 + chunk] = o["row_lse"]
        am[r0:r0 + chunk] = o["row_argmax"]
        tg[r0:r0 + chunk] = o["row_target"]
        s_num += o["s"] * o["n_valid"]
        ce_num += o["loss"] * o["n_valid"]
        nv += o["n_valid"]
        flags |= o["flags"] & oracle.FLAG_LABEL_RANGE
    orc = dict(s=s_num / nv, loss=ce_num / nv, n_valid=nv, flags=flags | (oracle.FLAG_EMPTY if nv == 0 else 0),
               row_lse=lse, row_argmax=am, row_target=tg,
               R_rows=oracle.residual(Zh[rows_R], y[rows_R])["R"])
    yield dict(w=w, Zd=Zd, Zh=Zh, y=y, yd=yd, res=res, g=g, orc=orc, rows_R=rows_R)
    del Zd, res
    torch.cuda.empty_cache()


def test_residual_full(lm):
    w, g, o, y = lm["w"], lm["g"], lm["orc"], lm["y"]
    log(f"[full] {w.name}: residual checks")
    assert int(g["n_valid"][0]) == o["n_valid"] and int(g["flags"][0]) == o["flags"]
    assert (g["row_argmax"] == o["row_argmax"]).all()
    Zh = lm["Zh"]
    assert (g["row_target"] == Zh[np.arange(w.N), y].astype(np.float32)).all()
    assert (np.abs(g["row_lse"] - o["row_lse"]) <= 1e-5 * np.maximum(1.0, np.abs(o["row_lse"]))).all()
    assert abs(float(g["loss"][0]) - o["loss"]) <= 1e-5 * max(1.0, abs(o["loss"]))
    cnt = np.bincount(y, minlength=w.V)[: w.V]
    cond = o["s"] + 2.0 * cnt / o["n_valid"]
    s = g["s"].astype(np.float64)
    assert rel_fro(s, o["s"]) <= 1e-5
    assert (np.abs(s - o["s"]) <= 1e-5 * cond + 1e-12).all()
    Ro = o["R_rows"]
    Rg = g["R_rows"]
    rows = lm["rows_R"]
    lab = np.zeros_like(Ro, dtype=bool)
    lab[np.arange(rows.size), y[rows]] = True
    assert (Rg[lab] <= 0).all() and (Rg[~lab] >= 0).all()
    assert (np.abs(Rg - Ro) <= (2.0 ** -8 + 1e-5) * np.abs(Ro) + 1e-5 * (Ro + lab) + 1e-30).all()


def test_head_vjp_full(lm):
    w, o, y, res = lm["w"], lm["orc"], lm["y"], lm["res"]
    N, d, V = w.N, w.d, w.V
    log(f"[full] {w.name}: head VJP")
    hb = synth.normal_bf16(N * d, synth.STREAM_H, 1.0)
    wb = synth.normal_bf16(d * V, synth.STREAM_W, 0.02)
    Hd, Wd = bf16_tensor(hb, (N, d)), bf16_tensor(wb, (d, V))
    Hh = synth.bf16_to_f32(hb).reshape(N, d)
    Wh = synth.bf16_to_f32(wb).reshape(d, V)
    q_prev = synth.normal_f32(V, synth.STREAM_U, 1e-4)
    q_prev = (q_prev - q_prev.astype(np.float64).mean()).astype(np.float32)
    t = 2
    q = torch.from_numpy(q_prev.copy()).to(dev())
    qh = bom.bom_ema(q, res["s"], w.beta1, t)
    out = bom.bom_head_vjp(Hd, Wd, res["R"], lm["yd"], qh, res["n_valid"], s=res["s"], lam=w.lam, want_db=True,
                           dh_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    _, qho = oracle.ema(q_prev, o["s"], f32(w.beta1), t)
    assert rel_fro(to_f64(qh), qho) <= 1e-5
    # 256 dW columns: spread over V, one in each of the last 96 tiles of 256 columns (the tiles a
    # partly filled last round of the wide kernel runs with split k), and the ragged last column;
    # 256 dH rows: spread over N (every 256-row tile) and the last row
    tiles_v = -(-V // 256)
    tail = [min(V - 1, t * 256 + (37 * t) % 256) for t in range(max(0, tiles_v - 96), tiles_v)]
    cols = np.unique(np.r_[np.linspace(0, V - 1, 256 - len(tail)).astype(int), tail, [V - 1]])
    rows = np.unique(np.r_[np.linspace(0, N - 1, 255).astype(int), [N - 1]])
    assert cols.size >= 250 and rows.size >= 250
    Zh = lm["Zh"]
    dWo = oracle.dW_cols_sub(Hh, Zh[:, cols], cols, V, y, o["row_lse"], qho, o["n_valid"], f32(w.lam))
    dHo = oracle.dH_rows_sub(Wh, Zh[rows], rows, y, o["row_lse"], qho, o["n_valid"], f32(w.lam))
    dWg = to_f64(out["dW"][:, torch.from_numpy(cols).to(dev())])
    dHg = to_f64(out["dH"][torch.from_numpy(rows).to(dev())])
    e_w, e_h = rel_fro(dWg, dWo), rel_fro(dHg, dHo)
    dbo = (1 - f32(w.lam)) * o["s"] + f32(w.lam) * qho
    e_b = rel_fro(to_f64(out["db"]), dbo)
    log(f"    rel err dW={e_w:.3e} dH={e_h:.3e} db={e_b:.3e}")
    assert e_w <= 2e-2 and e_h <= 2e-2 and e_b <= 1e-5
    # invariant over the whole matrix: every dW row sums to ~0 (rows of G sum to zero)
    rs = out["dW"].double().sum(1).cpu().numpy()
    ra = out["dW"].double().abs().sum(1).cpu().numpy()
    assert (np.abs(rs) <= 2e-2 * ra + 1e-12).all()
    del Hd, Wd, out
    torch.cuda.empty_cache()


def test_head_forward_full(lm):
    """The forward Z = H W at the full LM shapes (the blocked XCD order of its whole rounds at 32K, 1B and 8B):
    48 rows spread over every band of row tiles against the oracle, each element within two bf16 steps plus
    the fp32 accumulation error of its row; then the fused forward + residual on the same inputs: Z bitwise
    equal to the plain forward, row statistics on the sampled rows against the oracle run on that Z, and s,
    argmax, target, N_t and the flags against bom_residual on the same Z."""
    w, y = lm["w"], lm["y"]
    N, d, V = w.N, w.d, w.V
    log(f"[full] {w.name}: head forward")
    hb = synth.normal_bf16(N * d, synth.STREAM_H, 1.0)
    wb = synth.normal_bf16(d * V, synth.STREAM_W, 0.02)
    Hd, Wd = bf16_tensor(hb, (N, d)), bf16_tensor(wb, (d, V))
    Hh = synth.bf16_to_f32(hb).reshape(N, d).astype(np.float64)
    Wh = synth.bf16_to_f32(wb).reshape(d, V).astype(np.float64)
    del hb, wb
    Z = bom.bom_head_forward(Hd, Wd, None)
    torch.cuda.synchronize()
    rows = np.unique(np.r_[np.linspace(0, N - 1, 47).astype(int), [N - 1]])
    Zg = to_f64(Z[torch.from_numpy(rows).to(dev())])
    Zo = oracle.head_forward(Hh[rows], Wh, None)
    e = rel_fro(Zg, Zo)
    log(f"    forward rel err {e:.3e} on {rows.size} rows")
    assert e <= 2e-2
    acc = 1e-6 * (np.abs(Hh[rows]) @ np.abs(Wh))
    assert (np.abs(Zg - Zo) <= 2 * 2.0 ** -8 * np.abs(Zo) + acc + 1e-30).all()
    log(f"[full] {w.name}: fused forward + residual")
    fr = bom.bom_head_forward_residual(Hd, Wd, lm["yd"])
    torch.cuda.synchronize()
    assert torch.equal(fr["Z"].view(torch.int16), Z.view(torch.int16)), "fused Z differs from bom_head_forward"
    del Z
    ref = bom.bom_residual(fr["Z"], lm["yd"])
    torch.cuda.synchronize()
    for k in ("row_argmax", "row_target", "n_valid", "flags"):
        assert torch.equal(fr[k], ref[k]), k
    es = rel_fro(to_f64(fr["s"]), to_f64(ref["s"]))
    el = float((fr["row_lse"] - ref["row_lse"]).abs().max().item())
    log(f"    fused vs bom_residual: s rel {es:.2e}, max |lse diff| {el:.2e}")
    assert es <= 1e-5 and el <= 1e-5 * max(1.0, float(ref["row_lse"].abs().max().item()))
    o = oracle.residual(to_f64(fr["Z"][torch.from_numpy(rows).to(dev())]), y[rows], want_R=False)
    assert np.allclose(fr["row_lse"].cpu().numpy()[rows], o["row_lse"], rtol=1e-5, atol=1e-5)
    assert np.array_equal(fr["row_argmax"].cpu().numpy()[rows], o["row_argmax"])
    del fr, ref, Hd, Wd
    torch.cuda.empty_cache()


def _fill_seeded_(t, stream, std, start=0, chunk=1 << 27):
    n = t.numel()
    host = np.empty(min(chunk, n), np.float32)
    for s0 in range(0, n, chunk):
        m = min(chunk, n - s0)
        synth.normal_f32(m, stream, std, start=start + s0, out=host[:m])
        t[s0:s0 + m].copy_(torch.from_numpy(host[:m]))


@pytest.mark.parametrize("name", LM)
def test_update_full(name):
    w = BY_NAME[name]
    P = w.P
    log(f"[full] {name}: update over P={P} ({'factored' if w.factored else 'dense'})")
    theta = torch.empty(P, device=dev())
    u = torch.empty(P, device=dev())
    gen = torch.Generator(device=dev())
    gen.manual_seed(synth.BASE_SEED)
    # sampled regions come from the seeded generator (the oracle regenerates them); the rest is filled
    # on the device from torch's seeded generator with the same distribution
    theta.normal_(0.0, 0.02, generator=gen)
    u.normal_(0.0, 1e-3, generator=gen)
    if w.factored:
        bc, br = w.block_cols, w.block_rows
        nrows = -(-P // bc)
        nblocks = -(-nrows // br)
        blocks = [40, nblocks - 1]          # one interior block past the head slice, the short last block
        regions = []
        for b in blocks:
            e0 = b * br * bc
            e1 = min(P, (b + 1) * br * bc)
            regions.append((e0, e1))
    else:
        span = 1 << 20
        regions = [(P // 3, P // 3 + span), (P - span - 4, P)]
    for e0, e1 in regions:
        _fill_seeded_(theta[e0:e1], synth.STREAM_THETA, 0.02, start=e0)
        _fill_seeded_(u[e0:e1], synth.STREAM_U + 1, 1e-3, start=e0)
    th_before = theta.clone() if P <= 2_000_000_000 else None
    cfg = bom.make_update_cfg(lr=w.lr, beta2=w.beta2, eps=w.eps, t=1, lam=w.lam, factored=w.factored,
                              block_rows=w.block_rows, block_cols=w.block_cols)
    if w.factored:
        Rr = torch.zeros(nrows, device=dev())
        Cc = torch.zeros(nblocks * bc, device=dev())
        bom.bom_update(theta, Rr, u, cfg, v_col=Cc, segments=w.segments())
    else:
        v = torch.zeros(P, device=dev())
        bom.bom_update(theta, v, u, cfg, segments=w.segments())
    torch.cuda.synchronize()
    for e0, e1 in regions:
        th0 = synth.normal_f32(e1 - e0, synth.STREAM_THETA, 0.02, start=e0)
        u0 = synth.normal_f32(e1 - e0, synth.STREAM_U + 1, 1e-3, start=e0)
        if w.factored:
            b = e0 // (br * bc)
            r0, r1 = b * br, min(nrows, (b + 1) * br)
            tho, Ro, Co = oracle.update_factored(th0, np.zeros(r1 - r0), np.zeros(bc), u0, lr=f32(w.lr),
                                                 beta2=f32(w.beta2), eps=f32(w.eps), t=1, block_rows=br, block_cols=bc,
                                                 weight_decay=f32(w.weight_decay))
            assert rel_fro(to_f64(Rr[r0:r1]), Ro) <= 1e-5 and rel_fro(to_f64(Cc[b * bc:(b + 1) * bc]), Co) <= 1e-5
        else:
            tho, vo = oracle.update_dense(th0, np.zeros(e1 - e0), u0, lr=f32(w.lr), beta2=f32(w.beta2),
                                          eps=f32(w.eps), t=1, weight_decay=f32(w.weight_decay))
            assert (np.abs(to_f64(v[e0:e1]) - vo) <= 1e-5 * vo + 1e-30).all()
        err = np.abs(to_f64(theta[e0:e1]) - tho) / np.maximum(np.abs(tho), w.lr)
        log(f"    region [{e0}, {e1}): max rel err {err.max():.3e}")
        assert err.max() <= 1e-5
    if th_before is not None and not w.factored:
        # dense, t = 1: every element moves by at most lr (plus decay and one fp32 ulp)
        step = (theta.double() - (1 - w.lr * w.weight_decay) * th_before.double()).abs()
        assert float((step - w.lr - 2.5e-7 * th_before.double().abs()).max()) <= 0
    del theta, u
    torch.cuda.empty_cache()
