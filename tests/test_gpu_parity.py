"""GPU parity: every entry point of libbom.so against the fp64 oracle on the same seeded inputs.

Bars: bit-exact for argmax, the label-logit copy, N_t, flags and the sign pattern of R;
1e-5 relative for fp32 stages (s with a condition-aware per-element bound, lse, loss, q, q_hat,
db, theta, v and every fp32 GEMM); 2e-2 relative Frobenius for bf16-input GEMMs.
Sizes span several tiles and ragged tails; each case prints its name before touching the GPU.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import bf16_tensor, check_s, dev, gen_labels, gen_matrix, log, needs_gpu, rel_fro, to_f64
from paper_2609_36738_amd import bom

pytestmark = [pytest.mark.gpu, needs_gpu]

B1, B2, EPS, LAM = 0.9, 0.999, 1e-8, 0.5
f32 = lambda x: float(np.float32(x))  # the hyperparameter value the device actually uses


# ------------------------------------------------------------------------------------------------ residual
RESIDUAL_CASES = [
    # name, N, V, dtype, labels, ignore_frac, n_out_of_range, logit std
    ("tiny_f32_v10", 256, 10, "f32", "uniform", 0.0, 0, 0.23),
    ("bf16_v1000_ign", 300, 1000, "bf16", "uniform", 0.05, 4, 0.55),
    ("bf16_v1003_scalar", 77, 1003, "bf16", "zipf", 0.05, 2, 0.55),
    # register rows with more chunks per thread than the row holds (a chunk count from the fixed set): 2050
    # scalar columns at 512 threads need 5 chunks and run with 6, 10000 fp32 columns (float4) likewise
    ("bf16_v2050_scalar_spare_chunk", 300, 2050, "bf16", "zipf", 0.05, 2, 0.55),
    ("f32_v10000_spare_chunk", 64, 10000, "f32", "zipf", 0.05, 1, 0.55),
    ("f32_v4100_peaked", 129, 4100, "f32", "zipf", 0.05, 2, 11.0),
    ("bf16_v32000", 96, 32000, "bf16", "zipf", 0.05, 2, 0.55),
    ("bf16_v12000_multirow", 600, 12000, "bf16", "zipf", 0.05, 3, 0.55),
    ("bf16_v50304_packed", 64, 50304, "bf16", "zipf", 0.05, 2, 0.91),
    ("bf16_v50304_multirow", 600, 50304, "bf16", "zipf", 0.05, 3, 0.91),
    # split rows: parts of 1024 threads x 4 chunks (32,768 columns), up to 16 parts; wider rows take two passes
    ("bf16_v60000_split2", 40, 60000, "bf16", "zipf", 0.05, 2, 1.28),
    ("bf16_v70000_split3", 40, 70000, "bf16", "zipf", 0.05, 2, 1.28),
    ("bf16_v100008_split4", 24, 100008, "bf16", "zipf", 0.05, 2, 1.28),
    ("bf16_v128256_split4", 20, 128256, "bf16", "zipf", 0.05, 2, 1.28),
    # 64 row groups of 4 parts: three or four rows per group (the next row is prefetched during a row)
    ("bf16_v128256_split4_multirow", 200, 128256, "bf16", "zipf", 0.05, 3, 1.28),
    ("bf16_v200000_split7", 12, 200000, "bf16", "zipf", 0.05, 1, 1.28),
    ("bf16_v300000_split10", 8, 300000, "bf16", "zipf", 0.0, 1, 1.28),
    ("bf16_v330000_split11", 8, 330000, "bf16", "zipf", 0.0, 1, 1.28),
    ("bf16_v520000_split16", 6, 520000, "bf16", "zipf", 0.0, 1, 1.28),
    # 16 row groups of 16 parts with two or three rows each: the next rows' slices land in the LDS buffers
    ("bf16_v520000_split16_multirow", 40, 520000, "bf16", "zipf", 0.05, 2, 1.28),
    ("bf16_v530000_twopass", 4, 530000, "bf16", "zipf", 0.0, 1, 1.28),
    ("f32_v70003_twopass_scalar", 40, 70003, "f32", "zipf", 0.05, 2, 1.28),
    ("bf16_v4_n1", 1, 8, "bf16", "uniform", 0.0, 0, 1.0),
]


def _run_residual(Zd, yd, **kw):
    out = bom.bom_residual(Zd, yd, **kw)
    torch.cuda.synchronize()
    return out


def _compare_residual(name, Zh, y, out, orc, dtype):
    N, V = Zh.shape
    valid = (y != -100) & (y >= 0) & (y < V)
    assert int(out["n_valid"].item()) == orc["n_valid"] == int(valid.sum())
    assert int(out["flags"].item()) == orc["flags"]
    am = out["row_argmax"].cpu().numpy()
    assert (am == orc["row_argmax"]).all(), f"{name}: argmax"
    tg = out["row_target"].cpu().numpy()
    expect_tg = np.where(valid, Zh[np.arange(N), np.clip(y, 0, V - 1)], 0.0).astype(np.float32)
    assert (tg == expect_tg).all(), f"{name}: target copy"
    lse = to_f64(out["row_lse"])
    assert (np.abs(lse - orc["row_lse"]) <= 1e-5 * np.maximum(1.0, np.abs(orc["row_lse"]))).all(), f"{name}: lse"
    if orc["n_valid"] > 0:
        assert abs(out["loss"].item() - orc["loss"]) <= 1e-5 * max(1.0, abs(orc["loss"])), f"{name}: loss"
        cnt = np.bincount(y[valid], minlength=V)[:V]
        cond = orc["s"] + 2.0 * cnt / orc["n_valid"]          # mean_i (p_ij + [j = y_i]) over valid rows
        check_s(to_f64(out["s"]), orc, cond)
    R = to_f64(out["R"])
    Ro = orc["R"]
    # sign pattern: residual rows are <= 0 at the label and >= 0 elsewhere; ignored rows are 0
    lab = np.zeros_like(Ro, dtype=bool)
    lab[np.arange(N)[valid], y[valid]] = True
    assert (R[lab] <= 0).all() and (R[~lab] >= 0).all(), f"{name}: sign pattern"
    assert (R[~valid] == 0).all(), f"{name}: ignored rows"
    P = Ro + lab
    rtol = 2.0 ** -8 + 1e-5 if dtype == "bf16" else 1e-5
    assert (np.abs(R - Ro) <= rtol * np.abs(Ro) + 1e-5 * P + 1e-30).all(), f"{name}: R values"


@pytest.mark.parametrize("V", [1000, 12000, 32000, 50304])
def test_residual_argmax_ties(V):
    """Ties at the row maximum: the argmax is the first column holding it (a plain first-index
    argmax), whichever thread, chunk or wave the tied columns fall in; all-equal rows give 0."""
    N = 300
    log(f"[residual] argmax ties N={N} V={V}")
    Zh, _ = gen_matrix(N, V, synth.STREAM_Z, 0.55, "bf16")
    Zh = Zh.copy()
    rng = np.random.default_rng(1234 + V)
    for i in range(N):
        kind = i % 4
        if kind == 0:
            Zh[i, :] = 0.5                       # every column ties
        elif kind == 1:
            cols = rng.choice(V, size=3, replace=False)
            Zh[i, cols] = 8.0                    # three tied maxima anywhere in the row
        elif kind == 2:
            c0 = int(rng.integers(0, V - 8))
            Zh[i, c0] = Zh[i, c0 + 7] = 8.0      # tied maxima inside one 16-byte chunk
        else:
            Zh[i, V - 1] = Zh[i, V - 2] = 8.0    # tied maxima in the last chunk
    bits = (Zh.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    assert (synth.bf16_to_f32(bits).reshape(N, V) == Zh).all()
    Zd = bf16_tensor(bits, (N, V))
    y = gen_labels(N, V, "uniform")
    out = _run_residual(Zd, torch.from_numpy(y).to(dev()))
    am = out["row_argmax"].cpu().numpy()
    assert (am == np.argmax(Zh, axis=1)).all()
    assert (am[0::4] == 0).all()


@pytest.mark.parametrize("case", RESIDUAL_CASES, ids=[c[0] for c in RESIDUAL_CASES])
def test_residual_parity(case):
    name, N, V, dtype, kind, ign, oor, std = case
    log(f"[residual] {name} N={N} V={V} {dtype}")
    Zh, Zd = gen_matrix(N, V, synth.STREAM_Z, std, dtype)
    y = gen_labels(N, V, kind, ign, oor)
    yd = torch.from_numpy(y).to(dev())
    out = _run_residual(Zd, yd)
    orc = oracle.residual(Zh, y)
    _compare_residual(name, Zh, y, out, orc, dtype)
    # determinism: the same inputs give bitwise-identical outputs
    out2 = _run_residual(Zd, yd)
    for k in ("s", "row_lse", "R", "loss"):
        assert torch.equal(out[k], out2[k]), f"{name}: {k} not bitwise repeatable"


def test_residual_all_ignored_is_empty():
    log("[residual] all rows ignored")
    Zh, Zd = gen_matrix(50, 300, synth.STREAM_Z, 0.5, "bf16")
    y = np.full(50, -100, np.int32)
    out = _run_residual(Zd, torch.from_numpy(y).to(dev()))
    assert out["flags"].item() == bom.BOM_FLAG_EMPTY and out["n_valid"].item() == 0
    assert out["loss"].item() == 0 and (out["s"] == 0).all() and (out["R"].float() == 0).all()


# Z and R as views of wider buffers (leading dimensions past V) on each single-pass route: register rows,
# LDS-parked rows and split rows (four parts, several rows per row group); R's extra columns stay untouched.
@pytest.mark.parametrize("N,V,ldz,ldr,std", [(64, 1000, 1040, 1024, 0.5), (96, 50304, 50368, 50320, 0.91),
                                              (200, 128256, 128320, 128264, 1.28)],
                         ids=["register_rows", "lds_rows", "split_rows"])
def test_residual_strided_rows(N, V, ldz, ldr, std):
    log(f"[residual] strided Z and R views N={N} V={V} ldz={ldz} ldr={ldr}")
    Zh, Zd = gen_matrix(N, ldz, synth.STREAM_Z, std, "bf16")
    y = gen_labels(N, V, "zipf")
    Zv = Zd[:, :V]
    Rbuf = torch.full((N, ldr), 7.0, dtype=torch.bfloat16, device=dev())
    out = _run_residual(Zv, torch.from_numpy(y).to(dev()), R=Rbuf[:, :V])
    orc = oracle.residual(Zh[:, :V], y)
    out["R"] = Rbuf[:, :V]
    _compare_residual("strided", np.ascontiguousarray(Zh[:, :V]), y, out, orc, "bf16")
    assert (Rbuf[:, V:].float() == 7.0).all()


# ------------------------------------------------------------------------------------------------ EMA
def test_ema_parity():
    log("[ema] V=50304, 4 steps")
    V = 50304
    q = torch.zeros(V, device=dev())
    qo = np.zeros(V)
    for t in range(1, 5):
        s = synth.normal_f32(V, synth.STREAM_U + t, 1e-4)
        qh = bom.bom_ema(q, torch.from_numpy(s).to(dev()), B1, t)
        torch.cuda.synchronize()
        qo, qho = oracle.ema(qo, s, f32(B1), t)
        assert rel_fro(to_f64(q), qo) <= 1e-6 and rel_fro(to_f64(qh), qho) <= 1e-6


# ------------------------------------------------------------------------------------------------ head VJP
VJP_CASES = [
    # name, N, d, V, dtype, ignore_frac
    ("f32_tiny", 256, 128, 10, "f32", 0.0),
    ("f32_ragged", 130, 200, 520, "f32", 0.05),        # one launch (small fp32 heads)
    ("f32_simt_route", 600, 300, 700, "f32", 0.05),    # more than 64 tiles: the SIMT kernels with k splits
    ("bf16_ragged", 300, 136, 1000, "bf16", 0.05),
    ("bf16_unaligned_simt", 200, 64, 333, "bf16", 0.05),
    ("bf16_vision_head", 1024, 768, 1000, "bf16", 0.0),
    ("bf16_v4096", 512, 256, 4096, "bf16", 0.05),
    ("bf16_dH_splitk", 64, 128, 32000, "bf16", 0.0),
    ("bf16_tile256", 2048, 768, 4096, "bf16", 0.0),
    ("bf16_tile256_ragged_mnk", 2056, 520, 6000, "bf16", 0.05),
]


def _vjp_inputs(N, d, V, dtype, ign, t=3):
    Hh, Hd = gen_matrix(N, d, synth.STREAM_H, 1.0, dtype)
    Wh, Wd = gen_matrix(d, V, synth.STREAM_W, 0.02, dtype)
    Zh, Zd = gen_matrix(N, V, synth.STREAM_Z, math.sqrt(0.0004 * d), dtype)
    y = gen_labels(N, V, "zipf" if V > 1000 else "uniform", ign)
    # a task-space history is an EMA of zero-sum residual means, so it sums to zero too
    q_prev = synth.normal_f32(V, synth.STREAM_U, 0.01)
    q_prev = (q_prev - q_prev.astype(np.float64).mean()).astype(np.float32)
    return Hh, Hd, Wh, Wd, Zh, Zd, y, q_prev, t


@pytest.mark.parametrize("case", VJP_CASES, ids=[c[0] for c in VJP_CASES])
def test_head_vjp_parity(case):
    name, N, d, V, dtype, ign = case
    log(f"[head_vjp] {name} N={N} d={d} V={V} {dtype}")
    Hh, Hd, Wh, Wd, Zh, Zd, y, q_prev, t = _vjp_inputs(N, d, V, dtype, ign)
    yd = torch.from_numpy(y).to(dev())
    res = bom.bom_residual(Zd, yd)
    q = torch.from_numpy(q_prev.copy()).to(dev())
    qh = bom.bom_ema(q, res["s"], B1, t)
    g = bom.bom_head_vjp(Hd, Wd, res["R"], yd, qh, res["n_valid"], s=res["s"], lam=LAM, want_db=True,
                         dh_dtype=torch.float32)
    torch.cuda.synchronize()
    o = oracle.residual(Zh, y, want_R=False)
    _, qho = oracle.ema(q_prev, o["s"], f32(B1), t)
    dW = oracle.dW_cols(Hh, Zh, y, o["row_lse"], qho, o["n_valid"], LAM)
    dH = oracle.dH_rows(Wh, Zh, y, o["row_lse"], qho, o["n_valid"], LAM)
    db = oracle.db(Zh, y, o["row_lse"], qho, o["n_valid"], LAM)
    tol = 2e-2 if dtype == "bf16" else 1e-5
    e_dw, e_dh, e_db = rel_fro(to_f64(g["dW"]), dW), rel_fro(to_f64(g["dH"]), dH), rel_fro(to_f64(g["db"]), db)
    log(f"    rel err dW={e_dw:.3e} dH={e_dh:.3e} db={e_db:.3e}")
    assert e_dw <= tol and e_dh <= tol and e_db <= 1e-5
    # invariant: rows of G sum to zero, so dW 1 vanishes up to the rounding of G
    gdw = to_f64(g["dW"])
    assert (np.abs(gdw.sum(1)) <= (tol if dtype == "bf16" else 1e-4) * np.abs(gdw).sum(1) + 1e-12).all()


# d = 4096: 16 inner tiles per outer tile in both products, so their whole rounds run in the blocked XCD order
# (4 outer x 8 inner tiles per XCD round). dW's 47 outer tiles (ragged last) all run in whole rounds: XCDs 0-6
# own 6 of them (a group of 4, then one of 2) and XCD 7 owns 5 (4, then 1); dH runs 32 of its 41 outer tiles
# (ragged last) in whole rounds and the rest with split k. Sampled dW columns and dH rows include the ragged
# tiles and tiles of first and last groups.
XCD_COLS = np.r_[0:64, 5880:5940, 11700:11760, 11940:12000]
XCD_ROWS = np.r_[0:16, 5100:5120, 8180:8200, 10230:10248]


def test_head_vjp_blocked_xcd_order():
    N, d, V = 10248, 4096, 12000
    log(f"[head_vjp blocked XCD order] N={N} d={d} V={V}")
    Hh, Hd, Wh, Wd, Zh, Zd, y, q_prev, t = _vjp_inputs(N, d, V, "bf16", 0.05)
    yd = torch.from_numpy(y).to(dev())
    res = bom.bom_residual(Zd, yd)
    q = torch.from_numpy(q_prev.copy()).to(dev())
    qh = bom.bom_ema(q, res["s"], B1, t)
    g = bom.bom_head_vjp(Hd, Wd, res["R"], yd, qh, res["n_valid"], s=res["s"], lam=LAM, want_db=True,
                         dh_dtype=torch.float32)
    torch.cuda.synchronize()
    o = oracle.residual(Zh, y, want_R=False)
    _, qho = oracle.ema(q_prev, o["s"], f32(B1), t)
    dW = oracle.dW_cols(Hh, Zh, y, o["row_lse"], qho, o["n_valid"], LAM, cols=XCD_COLS)
    dH = oracle.dH_rows(Wh, Zh, y, o["row_lse"], qho, o["n_valid"], LAM, rows=XCD_ROWS)
    e_dw = rel_fro(to_f64(g["dW"])[:, XCD_COLS], dW)
    e_dh = rel_fro(to_f64(g["dH"])[XCD_ROWS], dH)
    log(f"    rel err dW={e_dw:.3e} dH={e_dh:.3e}")
    assert e_dw <= 2e-2 and e_dh <= 2e-2
    assert np.isfinite(to_f64(g["dW"])).all() and np.isfinite(to_f64(g["dH"])).all()


# Padded leading dimensions (multiples of 8) with V not a multiple of 8: the padding holds large values
# that must not reach any result (residual rows, s, dW, dH, db).
def test_head_vjp_padded_rows_ignore_padding():
    N, d, V, ld = 2048, 512, 4100, 4104
    log(f"[head_vjp padded] N={N} d={d} V={V} ld={ld}")
    Hh, Hd, Wh, Wd, Zh, Zd, y, q_prev, t = _vjp_inputs(N, d, V, "bf16", 0.05)
    def padded(x, rows):
        buf = torch.full((rows, ld), 1e4, dtype=torch.bfloat16, device=dev())
        buf[:, :V].copy_(x)
        return buf[:, :V]
    Zp, Wp = padded(Zd, N), padded(Wd, d)
    Rp = padded(torch.zeros((N, V), dtype=torch.bfloat16, device=dev()), N)
    yd = torch.from_numpy(y).to(dev())
    res = bom.bom_residual(Zp, yd, R=Rp)
    q = torch.from_numpy(q_prev.copy()).to(dev())
    qh = bom.bom_ema(q, res["s"], B1, t)
    g = bom.bom_head_vjp(Hd, Wp, Rp, yd, qh, res["n_valid"], s=res["s"], lam=LAM, want_db=True,
                         dh_dtype=torch.float32)
    torch.cuda.synchronize()
    assert float(Rp.storage_offset()) == 0 and torch.all(Rp.as_strided((N, ld), (ld, 1))[:, V:] == 1e4)
    o = oracle.residual(Zh, y, want_R=False)
    _, qho = oracle.ema(q_prev, o["s"], f32(B1), t)
    cols, rows = np.r_[0:32, V - 40:V], np.r_[0:16, N - 16:N]
    dW = oracle.dW_cols(Hh, Zh, y, o["row_lse"], qho, o["n_valid"], LAM, cols=cols)
    dH = oracle.dH_rows(Wh, Zh, y, o["row_lse"], qho, o["n_valid"], LAM, rows=rows)
    db = oracle.db(Zh, y, o["row_lse"], qho, o["n_valid"], LAM)
    e_s = rel_fro(to_f64(res["s"]), o["s"])
    e_dw, e_dh = rel_fro(to_f64(g["dW"])[:, cols], dW), rel_fro(to_f64(g["dH"])[rows], dH)
    e_db = rel_fro(to_f64(g["db"]), db)
    log(f"    rel err s={e_s:.3e} dW={e_dw:.3e} dH={e_dh:.3e} db={e_db:.3e}")
    assert e_s <= 1e-5 and e_dw <= 2e-2 and e_dh <= 2e-2 and e_db <= 1e-5


# More 256 x 256 output tiles than the chip has compute units: whole rounds run over the full k range
# and the leftover tiles split k (dW: the last column tiles; dH: the last row tiles), with ragged last
# tiles in both m and n and a k extent that is not a multiple of the 64-deep k tile.
ROUND_CASES = [
    # name, N, d, V; sampled dW columns and dH rows cover whole-round and leftover tiles and the ragged ends
    ("dW_leftover", 1032, 520, 24000, np.r_[0:40, 21700:21830, 23950:24000], np.r_[0:8, 1024:1032]),
    ("dH_leftover", 24600, 520, 2056, np.r_[0:16, 2040:2056], np.r_[0:32, 21740:21790, 24570:24600]),
]


# ldr = V + 4 (a leading dimension the MFMA tiles cannot stage): the same shapes on the SIMT kernels, whose
# own k splits must fit the workspace sized for the shape (regression: they once kept the wide plan's
# split count and wrote partials for every tile past the workspace).
# lam0: lambda = 0 (no history term: no rank-1 pre-pass, no rank-1 term in the epilogues or the split-k
# reduction), the plain cross-entropy backward of the AdamW arm.
@pytest.mark.parametrize("layout", ["dense", "ldr_plus4", "dense_lam0"])
@pytest.mark.parametrize("case", ROUND_CASES, ids=[c[0] for c in ROUND_CASES])
def test_head_vjp_whole_rounds_and_leftovers(case, layout):
    name, N, d, V, cols, rows = case
    lam = 0.0 if layout.endswith("lam0") else LAM
    log(f"[head_vjp] {name} N={N} d={d} V={V} R layout {layout} lambda {lam}")
    Hh, Hd, Wh, Wd, Zh, Zd, y, q_prev, t = _vjp_inputs(N, d, V, "bf16", 0.05)
    yd = torch.from_numpy(y).to(dev())
    R = None
    if layout == "ldr_plus4":
        R = torch.zeros((N, V + 4), dtype=torch.bfloat16, device=dev())[:, :V]
    res = bom.bom_residual(Zd, yd, R=R)
    q = torch.from_numpy(q_prev.copy()).to(dev())
    qh = bom.bom_ema(q, res["s"], B1, t)
    g = bom.bom_head_vjp(Hd, Wd, res["R"], yd, qh, res["n_valid"], s=res["s"], lam=lam, want_db=True,
                         dh_dtype=torch.float32)
    torch.cuda.synchronize()
    o = oracle.residual(Zh, y, want_R=False)
    _, qho = oracle.ema(q_prev, o["s"], f32(B1), t)
    dW = oracle.dW_cols(Hh, Zh, y, o["row_lse"], qho, o["n_valid"], lam, cols=cols)
    dH = oracle.dH_rows(Wh, Zh, y, o["row_lse"], qho, o["n_valid"], lam, rows=rows)
    gdw = to_f64(g["dW"])
    e_dw = rel_fro(gdw[:, cols], dW)
    e_dh = rel_fro(to_f64(g["dH"])[rows], dH)
    log(f"    rel err dW={e_dw:.3e} dH={e_dh:.3e}")
    assert e_dw <= 2e-2 and e_dh <= 2e-2
    assert np.isfinite(gdw).all() and np.isfinite(to_f64(g["dH"])).all()
    assert (np.abs(gdw.sum(1)) <= 2e-2 * np.abs(gdw).sum(1) + 1e-12).all()


# bf16 gradient storage: dW and db written as bf16 (formed in fp32, rounded once), on the fused
# small-product launch (vision head) and on the 256-tile route, with an accumulating dW_beta.
@pytest.mark.parametrize("N,d,V", [(1024, 768, 1000), (2048, 768, 4096)], ids=["fused_small", "tile256"])
def test_head_vjp_bf16_gradient_output(N, d, V):
    log(f"[head_vjp bf16 dW] N={N} d={d} V={V}")
    Hh, Hd, Wh, Wd, Zh, Zd, y, q_prev, t = _vjp_inputs(N, d, V, "bf16", 0.05)
    yd = torch.from_numpy(y).to(dev())
    res = bom.bom_residual(Zd, yd)
    q = torch.from_numpy(q_prev.copy()).to(dev())
    qh = bom.bom_ema(q, res["s"], B1, t)
    prev = oracle.round_bf16(synth.normal_f32(d * V, synth.STREAM_U, 1e-3).astype(np.float64))
    dW = torch.from_numpy(prev.view(np.int16)).view(torch.bfloat16).reshape(d, V).to(dev())
    db = torch.empty(V, dtype=torch.bfloat16, device=dev())
    g = bom.bom_head_vjp(Hd, Wd, res["R"], yd, qh, res["n_valid"], s=res["s"], lam=LAM, dW=dW, dW_beta=0.5, db=db,
                         want_db=True)
    torch.cuda.synchronize()
    o = oracle.residual(Zh, y, want_R=False)
    _, qho = oracle.ema(q_prev, o["s"], f32(B1), t)
    dWo = oracle.dW_cols(Hh, Zh, y, o["row_lse"], qho, o["n_valid"], LAM) + 0.5 * oracle.bf16_bits_to_f64(prev).reshape(d, V)
    dbo = oracle.db(Zh, y, o["row_lse"], qho, o["n_valid"], LAM)
    e_dw = rel_fro(to_f64(g["dW"]), dWo)
    log(f"    rel err dW={e_dw:.3e}")
    assert g["dW"].dtype == torch.bfloat16 and e_dw <= 2e-2
    # db is an fp32 stage rounded once to bf16: within one bf16 step of the rounded oracle value
    dbg = g["db"].cpu().view(torch.int16).numpy().view(np.uint16).astype(np.int32)
    assert (np.abs(dbg - oracle.round_bf16(dbo).astype(np.int32)) <= 1).all()


@pytest.mark.parametrize("lam", [0.0, 1.0, 0.25])
def test_head_vjp_tile256_lambda(lam):
    """Large-tile path at the edges of the mixture: lambda = 0 (plain cross-entropy backward),
    lambda = 1 (history only, the residual drops out of G) and an interior value."""
    N, d, V = 2048, 768, 4096
    log(f"[head_vjp] tile256 lambda={lam}")
    Hh, Hd, Wh, Wd, Zh, Zd, y, q_prev, t = _vjp_inputs(N, d, V, "bf16", 0.05)
    yd = torch.from_numpy(y).to(dev())
    res = bom.bom_residual(Zd, yd)
    q = torch.from_numpy(q_prev.copy()).to(dev())
    qh = bom.bom_ema(q, res["s"], B1, t)
    g = bom.bom_head_vjp(Hd, Wd, res["R"], yd, qh, res["n_valid"], lam=lam, dh_dtype=torch.float32)
    torch.cuda.synchronize()
    o = oracle.residual(Zh, y, want_R=False)
    _, qho = oracle.ema(q_prev, o["s"], f32(B1), t)
    cols = np.arange(0, V, 7)
    rows = np.arange(0, N, 5)
    dW = oracle.dW_cols(Hh, Zh, y, o["row_lse"], qho, o["n_valid"], f32(lam), cols=cols)
    dH = oracle.dH_rows(Wh, Zh, y, o["row_lse"], qho, o["n_valid"], f32(lam), rows=rows)
    e_dw = rel_fro(to_f64(g["dW"])[:, cols], dW)
    e_dh = rel_fro(to_f64(g["dH"])[rows], dH)
    log(f"    rel err dW={e_dw:.3e} dH={e_dh:.3e}")
    assert e_dw <= 2e-2 and e_dh <= 2e-2


@pytest.mark.parametrize("lam,want_dH", [(0.0, True), (1.0, True), (0.25, False)])
def test_head_vjp_small_fused_lambda(lam, want_dH):
    """Small products (one fused launch) at the edges of the mixture, on ragged tiles (d = 136), with
    and without dH; db checked too."""
    N, d, V = 300, 136, 1000
    log(f"[head_vjp] small fused lambda={lam} dH={want_dH}")
    Hh, Hd, Wh, Wd, Zh, Zd, y, q_prev, t = _vjp_inputs(N, d, V, "bf16", 0.05)
    yd = torch.from_numpy(y).to(dev())
    res = bom.bom_residual(Zd, yd)
    q = torch.from_numpy(q_prev.copy()).to(dev())
    qh = bom.bom_ema(q, res["s"], B1, t)
    g = bom.bom_head_vjp(Hd, Wd, res["R"], yd, qh, res["n_valid"], s=res["s"], lam=lam, want_db=True,
                         want_dH=want_dH, dh_dtype=torch.float32)
    torch.cuda.synchronize()
    o = oracle.residual(Zh, y, want_R=False)
    _, qho = oracle.ema(q_prev, o["s"], f32(B1), t)
    dW = oracle.dW_cols(Hh, Zh, y, o["row_lse"], qho, o["n_valid"], f32(lam))
    db = oracle.db(Zh, y, o["row_lse"], qho, o["n_valid"], f32(lam))
    e_dw, e_db = rel_fro(to_f64(g["dW"]), dW), rel_fro(to_f64(g["db"]), db)
    e_dh = 0.0
    if want_dH:
        e_dh = rel_fro(to_f64(g["dH"]), oracle.dH_rows(Wh, Zh, y, o["row_lse"], qho, o["n_valid"], f32(lam)))
    else:
        assert g.get("dH") is None
    log(f"    rel err dW={e_dw:.3e} dH={e_dh:.3e} db={e_db:.3e}")
    assert e_dw <= 2e-2 and e_dh <= 2e-2 and e_db <= 1e-5


def test_head_vjp_tile256_empty_batch():
    log("[head_vjp] tile256 N_t = 0")
    N, d, V = 2048, 768, 4096
    Hh, Hd, Wh, Wd, Zh, Zd, _, q_prev, t = _vjp_inputs(N, d, V, "bf16", 0.0)
    y = np.full(N, -100, np.int32)
    yd = torch.from_numpy(y).to(dev())
    res = bom.bom_residual(Zd, yd)
    g = bom.bom_head_vjp(Hd, Wd, res["R"], yd, torch.from_numpy(q_prev).to(dev()), res["n_valid"], lam=LAM)
    torch.cuda.synchronize()
    assert (g["dW"] == 0).all() and (g["dH"].float() == 0).all()


def test_head_vjp_bf16_dH_output_and_beta():
    log("[head_vjp] bf16 dH output, dW accumulation")
    N, d, V = 256, 128, 1000
    Hh, Hd, Wh, Wd, Zh, Zd, y, q_prev, t = _vjp_inputs(N, d, V, "bf16", 0.0)
    yd = torch.from_numpy(y).to(dev())
    res = bom.bom_residual(Zd, yd)
    q = torch.from_numpy(q_prev.copy()).to(dev())
    qh = bom.bom_ema(q, res["s"], B1, t)
    base = torch.full((d, V), 0.25, device=dev())
    g = bom.bom_head_vjp(Hd, Wd, res["R"], yd, qh, res["n_valid"], lam=LAM, dW=base.clone(), dW_beta=2.0)
    torch.cuda.synchronize()
    o = oracle.residual(Zh, y, want_R=False)
    _, qho = oracle.ema(q_prev, o["s"], f32(B1), t)
    dW = oracle.dW_cols(Hh, Zh, y, o["row_lse"], qho, o["n_valid"], LAM) + 0.5
    dH = oracle.dH_rows(Wh, Zh, y, o["row_lse"], qho, o["n_valid"], LAM)
    assert g["dH"].dtype == torch.bfloat16
    assert rel_fro(to_f64(g["dW"]), dW) <= 2e-2 and rel_fro(to_f64(g["dH"]), dH) <= 2e-2


def test_head_vjp_empty_batch_gives_zero():
    log("[head_vjp] N_t = 0")
    N, d, V = 64, 128, 256
    Hh, Hd, Wh, Wd, Zh, Zd, _, q_prev, t = _vjp_inputs(N, d, V, "bf16", 0.0)
    y = np.full(N, -100, np.int32)
    yd = torch.from_numpy(y).to(dev())
    res = bom.bom_residual(Zd, yd)
    qh = torch.from_numpy(q_prev).to(dev())
    g = bom.bom_head_vjp(Hd, Wd, res["R"], yd, qh, res["n_valid"], s=res["s"], want_db=True)
    torch.cuda.synchronize()
    assert (g["dW"] == 0).all() and (g["db"] == 0).all() and (g["dH"].float() == 0).all()


# ------------------------------------------------------------------------------------------------ telemetry
# Drift telemetry of the linear head over three steps with new features every step (so the own-step
# history drifts from the reprojection): M_W (and M_b) against the oracle after each step, the five
# statistics, and the fixed-feature case where there is no drift.
@pytest.mark.parametrize("N,d,V,dtype,bias,moving", [(1024, 768, 1000, "bf16", False, True),
                                                     (300, 136, 520, "f32", True, True),
                                                     (256, 64, 128, "bf16", True, False)],
                         ids=["vision_bf16", "ragged_f32_bias", "fixed_features"])
def test_head_telemetry_parity(N, d, V, dtype, bias, moving):
    log(f"[telemetry] N={N} d={d} V={V} {dtype} bias={bias} moving={moving}")
    MW = torch.zeros((d, V), device=dev())
    Mb = torch.zeros(V, device=dev()) if bias else None
    MWo, Mbo = np.zeros((d, V)), (np.zeros(V) if bias else None)
    q = torch.zeros(V, device=dev())
    qo = np.zeros(V)
    for t in range(1, 4):
        Hh, Hd = gen_matrix(N, d, synth.STREAM_H, 1.0, dtype, start=(t * N * d if moving else 0))
        Zh, Zd = gen_matrix(N, V, synth.STREAM_Z, 0.5, dtype, start=t * N * V)
        y = gen_labels(N, V, "uniform", 0.05)
        yd = torch.from_numpy(y).to(dev())
        res = bom.bom_residual(Zd, yd)
        qh = bom.bom_ema(q, res["s"], B1, t)
        tel = bom.bom_head_telemetry(Hd, res["R"], yd, res["s"], qh, res["n_valid"], MW, M_b=Mb, beta1=B1, t=t)
        torch.cuda.synchronize()
        # teacher forcing: the oracle step takes the GPU's own residual rows, s and q_hat
        R64, s64, qh64 = to_f64(res["R"]), to_f64(res["s"]), to_f64(qh)
        MWo, Mbo, st = oracle.head_telemetry(Hh, R64, y, s64, qh64, int(res["n_valid"].item()), MWo, Mbo,
                                             beta1=f32(B1), t=t)
        assert rel_fro(to_f64(MW), MWo) <= 1e-5
        if bias:
            assert rel_fro(to_f64(Mb), Mbo) <= 1e-5
        g = dict(zip(bom.TELEMETRY_FIELDS, tel["out"].cpu().numpy().astype(np.float64)))
        log("    " + " ".join(f"{k}={g[k]:.6f}/{st[k]:.6f}" for k in bom.TELEMETRY_FIELDS))
        for k in ("cos", "cancellation", "m_norm", "h_norm"):
            assert abs(g[k] - st[k]) <= 1e-5 * max(1.0, abs(st[k])), k
        assert abs(g["drift"] - st["drift"]) <= 1e-4 * max(1e-2, st["drift"])
        if not moving:
            assert g["drift"] <= 1e-4 and g["cos"] >= 1 - 1e-6


# ------------------------------------------------------------------------------------------------ forward
# The head forward in bf16 (row a0: the logits of the large workloads): matrix-core tiles with ragged m, n
# and k, the vision head with a bias, an LM shape checked on sampled rows (16 row tiles: the blocked XCD
# order, rows from four of them), and an unaligned shape on the
# SIMT kernel. Z is rounded once to bf16: the bar is the bf16-input GEMM bound, and every element within two
# bf16 steps plus the fp32 accumulation error of its row.
@pytest.mark.parametrize("N,d,V,bias,rows", [(2056, 520, 6000, False, None), (1024, 768, 1000, True, None),
                                            (4096, 768, 32000, False, np.r_[0:32, 1000:1040, 2300:2330, 4064:4096]),
                                            (300, 100, 333, True, None)],
                         ids=["tiles_ragged", "vision_bias", "lm_sampled", "simt_unaligned"])
def test_head_forward_bf16_parity(N, d, V, bias, rows):
    log(f"[forward bf16] N={N} d={d} V={V} bias={bias}")
    Hh, Hd = gen_matrix(N, d, synth.STREAM_H, 1.0, "bf16")
    Wh, Wd = gen_matrix(d, V, synth.STREAM_W, 0.02, "bf16")
    bh, bd = (gen_matrix(1, V, synth.STREAM_U, 0.1, "bf16") if bias else (None, None))
    Z = bom.bom_head_forward(Hd, Wd, None if bd is None else bd.reshape(V))
    torch.cuda.synchronize()
    sel = np.arange(N) if rows is None else rows
    Zo = oracle.head_forward(Hh[sel], Wh, None if bh is None else bh.reshape(V))
    Zg = to_f64(Z)[sel]
    assert Z.dtype == torch.bfloat16
    e = rel_fro(Zg, Zo)
    log(f"    rel err {e:.3e}")
    assert e <= 2e-2
    # element-wise: nearest bf16 of the exact value, give or take the fp32 accumulation of |H||W|
    acc = 1e-6 * (np.abs(Hh[sel]) @ np.abs(Wh))
    assert (np.abs(Zg - Zo) <= 2 * 2.0 ** -8 * np.abs(Zo) + acc + 1e-30).all()


# ------------------------------------------------------------------------------------------------ update
def _check_theta(th_gpu, th_o, lr, name):
    err = np.abs(th_gpu - th_o) / np.maximum(np.abs(th_o), lr)
    assert err.max() <= 1e-5, f"{name}: theta rel err {err.max():.3e}"


@pytest.mark.parametrize("split", [False, True], ids=["plain", "split"])
@pytest.mark.parametrize("offset", [0, 1], ids=["aligned", "misaligned"])
def test_update_dense_parity(split, offset):
    log(f"[update dense] split={split} offset={offset}")
    P = 1_000_003
    lr = 1e-3
    segs = [(0, 500_000, 0.01), (500_000, 3, 0.0)]
    th0 = synth.normal_f32(P, synth.STREAM_THETA, 0.02)
    buf_t = torch.zeros(P + offset, device=dev())
    buf_v = torch.zeros(P + offset, device=dev())
    theta, v = buf_t[offset:], buf_v[offset:]
    theta.copy_(torch.from_numpy(th0))
    tho, vo = th0.astype(np.float64), np.zeros(P)
    for t in range(1, 4):
        u = synth.normal_f32(P, synth.STREAM_U + t, 1e-3)
        h = synth.normal_f32(P, synth.STREAM_SPLIT_H + t, 1e-3) if split else None
        cfg = bom.make_update_cfg(lr=lr, beta2=B2, eps=EPS, t=t, lam=LAM)
        bom.bom_update(theta, v, torch.from_numpy(u).to(dev()), cfg, h=None if h is None else torch.from_numpy(h).to(dev()),
                       segments=segs, weight_decay=0.1)
        torch.cuda.synchronize()
        tho, vo = oracle.update_dense(tho, vo, u, lr=f32(lr), beta2=f32(B2), eps=f32(EPS), t=t, h=h, lam=f32(LAM),
                                      segments=[(a, b, f32(c)) for a, b, c in segs], weight_decay=f32(0.1))
        _check_theta(to_f64(theta), tho, lr, f"dense t={t}")
        vg = to_f64(v)
        assert (np.abs(vg - vo) <= 1e-5 * vo + 1e-30).all()


@pytest.mark.parametrize("br,bc,P", [(8, 64, 8 * 64 * 3 + 64 * 2 + 16), (4, 4096, 4096 * 9 + 2048), (3, 1024, 1024 * 7)],
                         ids=["bc64_ragged", "bc4096_ragged", "bc1024"])
def test_update_factored_parity(br, bc, P):
    log(f"[update factored] br={br} bc={bc} P={P}")
    lr = 1e-3
    nrows = -(-P // bc)
    nblocks = -(-nrows // br)
    th0 = synth.normal_f32(P, synth.STREAM_THETA, 0.02)
    theta = torch.from_numpy(th0.copy()).to(dev())
    Rr = torch.zeros(nrows, device=dev())
    Cc = torch.zeros(nblocks * bc, device=dev())
    tho, Ro, Co = th0.astype(np.float64), np.zeros(nrows), np.zeros(nblocks * bc)
    for t in range(1, 4):
        u = synth.normal_f32(P, synth.STREAM_U + t, 1e-3)
        cfg = bom.make_update_cfg(lr=lr, beta2=B2, eps=EPS, t=t, factored=True, block_rows=br, block_cols=bc)
        bom.bom_update(theta, Rr, torch.from_numpy(u).to(dev()), cfg, v_col=Cc, weight_decay=0.1)
        torch.cuda.synchronize()
        tho, Ro, Co = oracle.update_factored(tho, Ro, Co, u, lr=f32(lr), beta2=f32(B2), eps=f32(EPS), t=t,
                                             block_rows=br, block_cols=bc, weight_decay=f32(0.1))
        _check_theta(to_f64(theta), tho, lr, f"factored t={t}")
        assert rel_fro(to_f64(Rr), Ro) <= 1e-5 and rel_fro(to_f64(Cc), Co) <= 1e-5


# Global-norm clipping of the numerator (the device computes the norm; nothing returns to the host).
# u ~ N(0, 1e-3) over P = 10^6 has a norm near 1, so a threshold of 0.5 clips and 10 does not.
@pytest.mark.parametrize("clip,split,offset", [(0.5, True, 0), (0.5, False, 1), (10.0, False, 0)],
                         ids=["active_split_aligned", "active_plain_misaligned", "inactive"])
def test_update_dense_clip_parity(clip, split, offset):
    log(f"[update dense clip] clip={clip} split={split} offset={offset}")
    P = 1_000_003
    lr = 1e-3
    segs = [(0, 500_000, 0.01)]
    th0 = synth.normal_f32(P, synth.STREAM_THETA, 0.02)
    buf_t = torch.zeros(P + offset, device=dev())
    buf_v = torch.zeros(P + offset, device=dev())
    theta, v = buf_t[offset:], buf_v[offset:]
    theta.copy_(torch.from_numpy(th0))
    stats = torch.zeros(2, device=dev())
    tho, vo = th0.astype(np.float64), np.zeros(P)
    for t in range(1, 4):
        u = synth.normal_f32(P, synth.STREAM_U + t, 1e-3)
        h = synth.normal_f32(P, synth.STREAM_SPLIT_H + t, 1e-3) if split else None
        cfg = bom.make_update_cfg(lr=lr, beta2=B2, eps=EPS, t=t, lam=LAM, clip_norm=clip, clip_stats=stats)
        bom.bom_update(theta, v, torch.from_numpy(u).to(dev()), cfg, h=None if h is None else torch.from_numpy(h).to(dev()),
                       segments=segs, weight_decay=0.1)
        torch.cuda.synchronize()
        num = u.astype(np.float64) if h is None else (1 - f32(LAM)) * u.astype(np.float64) + f32(LAM) * h
        c_o = oracle.clip_factor(u, h=h, lam=f32(LAM), clip_norm=clip)
        norm_g, c_g = stats.cpu().numpy().astype(np.float64)
        assert abs(norm_g - np.linalg.norm(num)) <= 1e-5 * np.linalg.norm(num)
        assert abs(c_g - c_o) <= 1e-5 * c_o and (c_o < 1) == (clip < 1)
        tho, vo = oracle.update_dense(tho, vo, u, lr=f32(lr), beta2=f32(B2), eps=f32(EPS), t=t, h=h, lam=f32(LAM),
                                      segments=[(a, b, f32(c)) for a, b, c in segs], weight_decay=f32(0.1),
                                      clip_norm=clip)
        _check_theta(to_f64(theta), tho, lr, f"dense clip t={t}")
        vg = to_f64(v)
        assert (np.abs(vg - vo) <= 1e-5 * vo + 1e-30).all()


# Block-shared second moment (Adam-mini's map with the BOM numerator): segments tiling the buffer with
# per-element blocks (the dense kernels), one-wave blocks (up to 4096 elements, 16-byte or scalar accesses),
# long blocks in pieces (a block longer than its segment is the segment), ragged last blocks, and a
# misaligned layout whose segments start at odd offsets (scalar accesses throughout).
BLOCK_LAYOUTS = {
    "aligned": [(1000, 1, 0.0), (768 * 40 + 256, 768, 0.01), (4096 * 3, 4096, 0.01), (256 * 10, 256, 0.1),
                (45000, 20000, 0.01), (8192, 100000, 0.0), (49152 * 2 + 12, 49152, 0.01), (64, 64, 0.0)],
    "misaligned": [(1001, 1, 0.0), (700, 7, 0.01), (3001, 300, 0.1), (12345, 5000, 0.01), (4099, 4096, 0.0),
                   (9, 9, 0.0)],
}


@pytest.mark.parametrize("split,clip", [(False, 0.0), (True, 0.0), (False, 0.05)], ids=["plain", "split", "clip"])
@pytest.mark.parametrize("layout", list(BLOCK_LAYOUTS), ids=list(BLOCK_LAYOUTS))
def test_update_blocks_parity(layout, split, clip):
    spec = BLOCK_LAYOUTS[layout]
    segs, blocks, pos = [], [], 0
    for n, blk, wd in spec:
        segs.append((pos, n, wd))
        blocks.append(blk)
        pos += n
    P = pos
    nv = oracle.blocks_count(segs, blocks)
    log(f"[update blocks] {layout} split={split} clip={clip} P={P} blocks={nv}")
    lr = 1e-3
    th0 = synth.normal_f32(P, synth.STREAM_THETA, 0.02)
    theta = torch.from_numpy(th0.copy()).to(dev())
    v = torch.zeros(nv, device=dev())
    stats = torch.zeros(2, device=dev())
    tho, vo = th0.astype(np.float64), np.zeros(nv)
    segs32 = [(a, b, f32(c)) for a, b, c in segs]
    for t in range(1, 4):
        u = synth.normal_f32(P, synth.STREAM_U + t, 1e-3)
        u[:3] = 0.0      # a zero block inside the first segment
        h = synth.normal_f32(P, synth.STREAM_SPLIT_H + t, 1e-3) if split else None
        cfg = bom.make_update_cfg(lr=lr, beta2=B2, eps=EPS, t=t, lam=LAM, clip_norm=clip, clip_stats=stats,
                                  blocks=blocks)
        bom.bom_update(theta, v, torch.from_numpy(u).to(dev()), cfg, segments=segs,
                       h=None if h is None else torch.from_numpy(h).to(dev()))
        torch.cuda.synchronize()
        tho, vo = oracle.update_blocks(tho, vo, u, lr=f32(lr), beta2=f32(B2), eps=f32(EPS), t=t, segments=segs32,
                                       blocks=blocks, h=h, lam=f32(LAM), clip_norm=clip)
        _check_theta(to_f64(theta), tho, lr, f"blocks {layout} t={t}")
        vg = to_f64(v)
        assert (np.abs(vg - vo) <= 1e-5 * vo + 1e-30).all(), f"blocks {layout} t={t}: v"
        if clip:
            assert abs(float(stats[1]) - oracle.clip_factor(u, h=h, lam=f32(LAM), clip_norm=clip)) <= 1e-5


@pytest.mark.parametrize("br,bc,P,clip", [(4, 4096, 4096 * 9 + 2048, 0.1), (8, 64, 8 * 64 * 3 + 64 * 2 + 16, 0.02)],
                         ids=["bc4096_rows", "bc64_strips"])
def test_update_factored_clip_parity(br, bc, P, clip):
    log(f"[update factored clip] br={br} bc={bc} P={P} clip={clip}")
    lr = 1e-3
    nrows = -(-P // bc)
    nblocks = -(-nrows // br)
    th0 = synth.normal_f32(P, synth.STREAM_THETA, 0.02)
    theta = torch.from_numpy(th0.copy()).to(dev())
    Rr = torch.zeros(nrows, device=dev())
    Cc = torch.zeros(nblocks * bc, device=dev())
    stats = torch.zeros(2, device=dev())
    tho, Ro, Co = th0.astype(np.float64), np.zeros(nrows), np.zeros(nblocks * bc)
    for t in range(1, 4):
        u = synth.normal_f32(P, synth.STREAM_U + t, 1e-3)
        cfg = bom.make_update_cfg(lr=lr, beta2=B2, eps=EPS, t=t, factored=True, block_rows=br, block_cols=bc,
                                  clip_norm=clip, clip_stats=stats)
        bom.bom_update(theta, Rr, torch.from_numpy(u).to(dev()), cfg, v_col=Cc, weight_decay=0.1)
        torch.cuda.synchronize()
        c_o = oracle.clip_factor(u, clip_norm=clip)
        norm_g, c_g = stats.cpu().numpy().astype(np.float64)
        assert c_o < 1 and abs(c_g - c_o) <= 1e-5 * c_o
        assert abs(norm_g - np.linalg.norm(u.astype(np.float64))) <= 1e-5 * np.linalg.norm(u.astype(np.float64))
        tho, Ro, Co = oracle.update_factored(tho, Ro, Co, u, lr=f32(lr), beta2=f32(B2), eps=f32(EPS), t=t,
                                             block_rows=br, block_cols=bc, weight_decay=f32(0.1), clip_norm=clip)
        _check_theta(to_f64(theta), tho, lr, f"factored clip t={t}")
        assert rel_fro(to_f64(Rr), Ro) <= 1e-5 and rel_fro(to_f64(Cc), Co) <= 1e-5


def _bf16_dev(bits, offset=0):
    buf = torch.zeros(bits.size + offset, dtype=torch.bfloat16, device=dev())
    out = buf[offset:]
    out.copy_(torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16))
    return out


def _bits(t):
    return t.cpu().view(torch.int16).numpy().view(np.uint16)


def _check_bf16(g, o, name, min_exact=0.999, floor=None):
    """bf16 results against the oracle's once-rounded fp64 step: at most one bf16 step apart (the kernel
    rounds its fp32 result, the oracle its fp64 result, so a value within an fp32 rounding of a bf16
    midpoint may land on the other side), and bitwise equal almost everywhere. `floor` bounds the
    absolute fp32 error of results formed by cancellation (theta - step near zero), where it can
    exceed one bf16 step of the tiny result."""
    gi, oi = g.astype(np.int32), o.astype(np.int32)
    same_sign = (gi >> 15) == (oi >> 15)
    ok = same_sign & (np.abs(gi - oi) <= 1) | ((gi & 0x7FFF) == 0) & ((oi & 0x7FFF) <= 1)
    if floor is not None:
        ok |= np.abs(oracle.bf16_bits_to_f64(g) - oracle.bf16_bits_to_f64(o)) <= floor
    if not ok.all():
        bad = np.flatnonzero(~ok)[:8]
        gv, ov = oracle.bf16_bits_to_f64(g[bad]), oracle.bf16_bits_to_f64(o[bad])
        raise AssertionError(f"{name}: {(~ok).sum()} elements beyond one bf16 step, e.g. "
                             + ", ".join(f"[{i}] gpu {a:.6e} ({x:#06x}) oracle {b:.6e} ({y:#06x})"
                                         for i, a, b, x, y in zip(bad, gv, ov, g[bad], o[bad])))
    assert (gi == oi).mean() >= min_exact, f"{name}: bitwise-equal fraction {(gi == oi).mean():.5f}"


# bf16 state storage (theta, v, u, h bf16; fp32 arithmetic; theta and v rounded to nearest-even bf16).
@pytest.mark.parametrize("split,offset,clip", [(False, 0, 0.0), (True, 1, 0.0), (False, 0, 0.5)],
                         ids=["plain_aligned", "split_misaligned", "clipped"])
def test_update_dense_bf16_parity(split, offset, clip):
    log(f"[update dense bf16] split={split} offset={offset} clip={clip}")
    P = 1_000_003
    lr = 1e-3
    segs = [(0, 500_000, 0.01), (500_000, 3, 0.0)]
    tb = oracle.round_bf16(synth.normal_f32(P, synth.STREAM_THETA, 0.02).astype(np.float64))
    vb = np.zeros(P, np.uint16)
    theta, v = _bf16_dev(tb, offset), _bf16_dev(vb, offset)
    for t in range(1, 4):
        ub = oracle.round_bf16(synth.normal_f32(P, synth.STREAM_U + t, 1e-3).astype(np.float64))
        hb = oracle.round_bf16(synth.normal_f32(P, synth.STREAM_SPLIT_H + t, 1e-3).astype(np.float64)) if split else None
        cfg = bom.make_update_cfg(lr=lr, beta2=B2, eps=EPS, t=t, lam=LAM, clip_norm=clip, state_dtype=torch.bfloat16)
        bom.bom_update(theta, v, _bf16_dev(ub, offset), cfg, h=None if hb is None else _bf16_dev(hb, offset),
                       segments=segs, weight_decay=0.1)
        torch.cuda.synchronize()
        # fp32 absolute error of theta - step: a few units of 2^-24 of the operands (theta and lr * ratio)
        floor = 1e-6 * (np.abs(oracle.bf16_bits_to_f64(tb)) + lr)
        tb, vb = oracle.update_dense_bf16(tb, vb, ub, h_bits=hb, lr=f32(lr), beta2=f32(B2), eps=f32(EPS), t=t,
                                          lam=f32(LAM), segments=[(a, b, f32(c)) for a, b, c in segs],
                                          weight_decay=f32(0.1), clip_norm=clip)
        _check_bf16(_bits(theta), tb, f"theta t={t}", floor=floor)
        _check_bf16(_bits(v), vb, f"v t={t}")
        # teacher forcing: the next step starts from the GPU's own state
        tb, vb = _bits(theta), _bits(v)


# ------------------------------------------------------------------------------------------------ loop
def test_tiny_classifier_20_steps():
    """Ten-class linear softmax classifier (N = 256, d = 128), 20 BOM steps entirely on the GPU
    (forward, residual, EMA, head VJP into the flat u, update). Every step is teacher-forced: the oracle
    takes the GPU's theta, v and q from before the step, and the GPU's results after it must match at the
    fp32 bound (1e-5). A second oracle trajectory runs free from the same start and bounds the drift."""
    log("[loop] tiny classifier, 20 steps")
    N, d, V = 256, 128, 10
    P = d * V + V
    lr, wd = 1e-2, 0.01
    H = synth.normal_f32(N * d, synth.STREAM_H, 1.0).reshape(N, d)
    y = synth.labels_uniform(N, V)
    th0 = np.concatenate([synth.normal_f32(d * V, synth.STREAM_W, 0.02), np.zeros(V, np.float32)])
    segs = [(0, d * V, wd), (d * V, V, 0.0)]
    Hd, yd = torch.from_numpy(H).to(dev()), torch.from_numpy(y).to(dev())
    theta = torch.from_numpy(th0.copy()).to(dev())
    v = torch.zeros(P, device=dev())
    u = torch.zeros(P, device=dev())
    q = torch.zeros(V, device=dev())
    tho, vo, qo = th0.astype(np.float64), np.zeros(P), np.zeros(V)
    worst = 0.0
    seg32 = [(a, b_, f32(c)) for a, b_, c in segs]
    for t in range(1, 21):
        th_in, v_in, q_in = to_f64(theta), to_f64(v), to_f64(q)
        W = theta[: d * V].view(d, V)
        b = theta[d * V:]
        Z = bom.bom_head_forward(Hd, W, b)
        res = bom.bom_residual(Z, yd)
        qh = bom.bom_ema(q, res["s"], B1, t)
        bom.bom_head_vjp(Hd, W, res["R"], yd, qh, res["n_valid"], s=res["s"], lam=LAM, dW=u[: d * V].view(d, V),
                         db=u[d * V:], want_dH=False)
        bom.bom_update(theta, v, u, bom.make_update_cfg(lr=lr, beta2=B2, eps=EPS, t=t, lam=LAM), segments=segs)
        torch.cuda.synchronize()
        # teacher-forced step from the GPU's own state: the fp32 bound
        tf = oracle.bom_step_linear_head(H, y, th_in, v_in, q_in, t, d=d, V=V, lr=f32(lr), lam=f32(LAM),
                                         beta1=f32(B1), beta2=f32(B2), eps=f32(EPS), segments=seg32)
        thg, vg, ug = to_f64(theta), to_f64(v), to_f64(u)
        assert rel_fro(to_f64(q), tf["q"]) <= 1e-5, f"step {t}: q"
        assert rel_fro(to_f64(qh), tf["q_hat"]) <= 1e-5, f"step {t}: q_hat"
        assert rel_fro(ug, tf["u"]) <= 1e-5, f"step {t}: u = (dW, db)"
        # the update stage on its own input (the GPU's u): theta and v per element
        tho_u, vo_u = oracle.update_dense(th_in, v_in, ug, lr=f32(lr), beta2=f32(B2), eps=f32(EPS), t=t,
                                          segments=seg32)
        err_t = np.max(np.abs(thg - tho_u) / np.maximum(np.abs(tho_u), lr))
        assert err_t <= 1e-5, f"step {t}: theta rel err {err_t:.3e}"
        assert (np.abs(vg - vo_u) <= 1e-5 * vo_u + 1e-30).all(), f"step {t}: v"
        # free-running oracle trajectory: drift of the GPU's trajectory from it
        st = oracle.bom_step_linear_head(H, y, tho, vo, qo, t, d=d, V=V, lr=f32(lr), lam=f32(LAM), beta1=f32(B1),
                                         beta2=f32(B2), eps=f32(EPS), segments=seg32)
        tho, vo, qo = st["theta"], st["v"], st["q"]
        worst = max(worst, np.max(np.abs(thg - tho) / np.maximum(np.abs(tho), lr)))
    log(f"    max relative theta deviation over 20 free-running steps: {worst:.3e}")
    assert worst <= 1e-3


# ------------------------------------------------------------------------------------------------ full size
def test_vision_head_full_size():
    """1000-class head: N = 1024, d = 768, V = 1000, flat P = 86M; every stage at full size,
    in the launch configuration the benchmark times, checked in full against the oracle."""
    log("[full] vision head c1000, P=86M")
    N, d, V, P = 1024, 768, 1000, 86_000_000
    lr = 3e-5
    Hh, Hd, Wh, Wd, Zh, Zd, y, q_prev, _ = _vjp_inputs(N, d, V, "bf16", 0.0)
    y = synth.labels_uniform(N, V)
    yd = torch.from_numpy(y).to(dev())
    res = bom.bom_residual(Zd, yd)
    q = torch.zeros(V, device=dev())
    qh = bom.bom_ema(q, res["s"], B1, 1)
    theta = torch.from_numpy(synth.normal_f32(P, synth.STREAM_THETA, 0.02)).to(dev())
    u = torch.from_numpy(synth.normal_f32(P, synth.STREAM_U + 1, 1e-3)).to(dev())
    v = torch.zeros(P, device=dev())
    g = bom.bom_head_vjp(Hd, Wd, res["R"], yd, qh, res["n_valid"], lam=LAM, dW=u[: d * V].view(d, V),
                         dh_dtype=torch.bfloat16)
    u_head = to_f64(u[: d * V])
    bom.bom_update(theta, v, u, bom.make_update_cfg(lr=lr, beta2=B2, eps=EPS, t=1, lam=LAM), weight_decay=0.01)
    torch.cuda.synchronize()
    o = oracle.residual(Zh, y)
    _compare_residual("vision_full", Zh, y, res, o, "bf16")
    _, qho = oracle.ema(np.zeros(V), o["s"], f32(B1), 1)
    assert rel_fro(to_f64(qh), qho) <= 1e-5
    dW = oracle.dW_cols(Hh, Zh, y, o["row_lse"], qho, o["n_valid"], LAM)
    dH = oracle.dH_rows(Wh, Zh, y, o["row_lse"], qho, o["n_valid"], LAM)
    assert rel_fro(u_head.reshape(d, V), dW) <= 2e-2 and rel_fro(to_f64(g["dH"]), dH) <= 2e-2
    # update: the backbone slice holds seeded u, so the oracle takes the generator's values there; the head
    # slice holds the GPU's dW, which the oracle takes as its u there (teacher forcing on the update's input)
    th_in = synth.normal_f32(P, synth.STREAM_THETA, 0.02)
    u_in = synth.normal_f32(P, synth.STREAM_U + 1, 1e-3).astype(np.float64)
    u_in[: d * V] = u_head
    tho, vo = oracle.update_dense(th_in, np.zeros(P), u_in, lr=f32(lr), beta2=f32(B2), eps=f32(EPS), t=1,
                                  weight_decay=f32(0.01))
    _check_theta(to_f64(theta), tho, lr, "vision theta (head slice from the GPU's dW, backbone seeded)")
    assert (np.abs(to_f64(v) - vo) <= 1e-5 * vo + 1e-30).all()


# ------------------------------------------------------------------------------------------------ head VJP from Z
# The logits input (is_residual = 0): the kernels form R from Z and row_lse as their operand copies pass
# through registers. Every kernel route: SIMT (fp32, and bf16 with an unaligned V), the fused small-product
# launch, the 128-tile kernels that fold G while staging (k above 8192), the 256-tile pair launch and the
# separate 256-tile launches with leftover split-k tiles. Each is checked against the oracle (which has
# no R input at all) and against the same products from the stored R (equal up to one rounding of R).
Z_CASES = [
    # name, N, d, V, dtype, ignore_frac, out-of-range labels, sampled dW columns, sampled dH rows (None: all)
    ("f32_tiny", 256, 128, 10, "f32", 0.05, 2, None, None),
    ("bf16_unaligned_simt", 200, 64, 333, "bf16", 0.05, 2, None, None),
    ("bf16_fused_small", 1024, 768, 1000, "bf16", 0.05, 2, None, None),
    ("bf16_fold128", 64, 128, 32000, "bf16", 0.05, 2, None, None),
    ("bf16_pair", 4096, 768, 32000, "bf16", 0.05, 2, np.r_[0:64, 31900:32000], np.r_[0:32, 4064:4096]),
    ("bf16_dW_leftover", 1032, 520, 24000, "bf16", 0.05, 0, np.r_[0:40, 21700:21830, 23950:24000],
     np.r_[0:8, 1024:1032]),
    ("bf16_dH_leftover", 24600, 520, 2056, "bf16", 0.05, 0, np.r_[0:16, 2040:2056],
     np.r_[0:32, 21740:21790, 24570:24600]),
]


@pytest.mark.parametrize("case", Z_CASES, ids=[c[0] for c in Z_CASES])
def test_head_vjp_from_logits(case):
    name, N, d, V, dtype, ign, noor, cols, rows = case
    log(f"[head_vjp from Z] {name} N={N} d={d} V={V} {dtype}")
    Hh, Hd, Wh, Wd, Zh, Zd, _, q_prev, t = _vjp_inputs(N, d, V, dtype, ign)
    y = gen_labels(N, V, "zipf" if V > 1000 else "uniform", ign, noor)
    yd = torch.from_numpy(y).to(dev())
    res = bom.bom_residual(Zd, yd)
    q = torch.from_numpy(q_prev.copy()).to(dev())
    qh = bom.bom_ema(q, res["s"], B1, t)
    kw = dict(s=res["s"], lam=LAM, want_db=True, dh_dtype=torch.float32)
    gz = bom.bom_head_vjp(Hd, Wd, Zd, yd, qh, res["n_valid"], row_lse=res["row_lse"], **kw)
    gr = bom.bom_head_vjp(Hd, Wd, res["R"], yd, qh, res["n_valid"], **kw)
    torch.cuda.synchronize()
    o = oracle.residual(Zh, y, want_R=False)
    _, qho = oracle.ema(q_prev, o["s"], f32(B1), t)
    cols = np.arange(V) if cols is None else cols
    rows = np.arange(N) if rows is None else rows
    dW = oracle.dW_cols(Hh, Zh, y, o["row_lse"], qho, o["n_valid"], LAM, cols=cols)
    dH = oracle.dH_rows(Wh, Zh, y, o["row_lse"], qho, o["n_valid"], LAM, rows=rows)
    db = oracle.db(Zh, y, o["row_lse"], qho, o["n_valid"], LAM)
    tol = 2e-2 if dtype == "bf16" else 1e-5
    zw, zh = to_f64(gz["dW"]), to_f64(gz["dH"])
    e_dw, e_dh, e_db = rel_fro(zw[:, cols], dW), rel_fro(zh[rows], dH), rel_fro(to_f64(gz["db"]), db)
    # from Z against from the stored R: R formed in the kernels and R written by bom_residual agree up to
    # one rounding of R in some elements
    d_w, d_h = rel_fro(zw, to_f64(gr["dW"])), rel_fro(zh, to_f64(gr["dH"]))
    log(f"    rel err dW={e_dw:.3e} dH={e_dh:.3e} db={e_db:.3e}; Z vs R route dW={d_w:.2e} dH={d_h:.2e}")
    assert e_dw <= tol and e_dh <= tol and e_db <= 1e-5
    assert d_w <= (4e-3 if dtype == "bf16" else 1e-6) and d_h <= (4e-3 if dtype == "bf16" else 1e-6)
    assert np.isfinite(zw).all() and np.isfinite(zh).all()
    # rows outside I contribute nothing: their dH rows are the rank-1 term's zero rows
    bad = np.flatnonzero((y < 0) | (y >= V))
    assert (zh[bad] == 0).all()


# ------------------------------------------------------------------------------------------------ AdamW arm
# The comparison optimizer of the cost model: AdamW with its dense first moment, dense or factored second
# moment, three steps teacher-forced (each step starts from the GPU's own state).
@pytest.mark.parametrize("offset", [0, 1], ids=["aligned", "misaligned"])
def test_adamw_dense_parity(offset):
    log(f"[adamw dense] offset={offset}")
    P, lr, b1 = 1_000_003, 1e-3, 0.9
    segs = [(0, 500_000, 0.01), (500_000, 3, 0.0)]
    th = synth.normal_f32(P, synth.STREAM_THETA, 0.02)
    buf = lambda x: torch.from_numpy(np.r_[np.zeros(offset, np.float32), x.astype(np.float32)]).to(dev())[offset:]
    theta, m, v = buf(th), buf(np.zeros(P)), buf(np.zeros(P))
    for t in range(1, 4):
        g = synth.normal_f32(P, synth.STREAM_U + t, 1e-3)
        th_in, m_in, v_in = to_f64(theta), to_f64(m), to_f64(v)
        cfg = bom.make_update_cfg(lr=lr, beta2=B2, eps=EPS, t=t, u_scale=0.5)
        bom.bom_adamw_update(theta, m, v, buf(g), cfg, beta1=b1, segments=segs, weight_decay=0.1)
        torch.cuda.synchronize()
        tho, mo, vo = oracle.update_adamw(th_in, m_in, v_in, g, lr=f32(lr), beta1=f32(b1), beta2=f32(B2),
                                          eps=f32(EPS), t=t, segments=[(a, b_, f32(c)) for a, b_, c in segs],
                                          weight_decay=f32(0.1), u_scale=0.5)
        _check_theta(to_f64(theta), tho, lr, f"adamw theta t={t}")
        # m = b1 m + (1 - b1) g cancels: the bound is relative to the magnitude of its terms
        scale_m = b1 * np.abs(m_in) + (1 - b1) * 0.5 * np.abs(g.astype(np.float64))
        assert (np.abs(to_f64(m) - mo) <= 1e-5 * scale_m + 1e-30).all(), f"m t={t}"
        assert (np.abs(to_f64(v) - vo) <= 1e-5 * vo + 1e-30).all(), f"v t={t}"


@pytest.mark.parametrize("bc", [1024, 4096])
def test_adamw_factored_parity(bc):
    log(f"[adamw factored] block_cols={bc}")
    br, lr, b1 = 64, 1e-3, 0.9
    P = 3 * br * bc + 7 * bc + 1000   # three whole blocks, a short last block, a short last row
    nrows = -(-P // bc)
    nblocks = -(-nrows // br)
    theta = torch.from_numpy(synth.normal_f32(P, synth.STREAM_THETA, 0.02)).to(dev())
    m = torch.zeros(P, device=dev())
    Rr, Cc = torch.zeros(nrows, device=dev()), torch.zeros(nblocks * bc, device=dev())
    for t in range(1, 4):
        g = synth.normal_f32(P, synth.STREAM_U + t, 1e-3)
        th_in, m_in, R_in, C_in = to_f64(theta), to_f64(m), to_f64(Rr), to_f64(Cc)
        cfg = bom.make_update_cfg(lr=lr, beta2=B2, eps=EPS, t=t, factored=True, block_rows=br, block_cols=bc)
        bom.bom_adamw_update(theta, m, Rr, torch.from_numpy(g).to(dev()), cfg, beta1=b1, v_col=Cc, weight_decay=0.1)
        torch.cuda.synchronize()
        tho, mo, Ro, Co = oracle.update_adamw_factored(th_in, m_in, R_in, C_in, g, lr=f32(lr), beta1=f32(b1),
                                                       beta2=f32(B2), eps=f32(EPS), t=t, block_rows=br,
                                                       block_cols=bc, weight_decay=f32(0.1))
        _check_theta(to_f64(theta), tho, lr, f"adamw factored theta t={t}")
        assert rel_fro(to_f64(Rr), Ro) <= 1e-5 and rel_fro(to_f64(Cc), Co) <= 1e-5
        scale_m = b1 * np.abs(m_in) + (1 - b1) * np.abs(g.astype(np.float64))
        assert (np.abs(to_f64(m) - mo) <= 1e-5 * scale_m + 1e-30).all(), f"m t={t}"


# ------------------------------------------------------------------------------------------------ forward + residual
# bom_head_forward_residual: Z = H W (+ b), then the residual of that Z, with the row statistics reduced in
# the forward's epilogue (per 256-column tile) on the matrix-core path. Z must equal bom_head_forward's
# bitwise; every residual output is checked against the oracle on the GPU's own Z, and the integer outputs
# against bom_residual on it.
FWD_RES_CASES = [
    # name, N, d, V, dtype, bias, ignore_frac, out-of-range labels
    ("bf16_ragged_tiles", 300, 136, 1000, "bf16", True, 0.05, 2),
    ("bf16_lm_32k", 512, 768, 32000, "bf16", False, 0.05, 2),
    ("bf16_v128k", 64, 256, 128256, "bf16", False, 0.0, 0),
    ("bf16_unaligned_v", 200, 64, 333, "bf16", False, 0.05, 2),
    ("f32_tiny", 256, 128, 10, "f32", True, 0.0, 0),
]


@pytest.mark.parametrize("case", FWD_RES_CASES, ids=[c[0] for c in FWD_RES_CASES])
def test_head_forward_residual_parity(case):
    name, N, d, V, dtype, with_bias, ign, noor = case
    log(f"[forward+residual] {name} N={N} d={d} V={V} {dtype} bias={with_bias}")
    Hh, Hd = gen_matrix(N, d, synth.STREAM_H, 1.0, dtype)
    Wh, Wd = gen_matrix(d, V, synth.STREAM_W, 0.02, dtype)
    bd = None
    if with_bias:
        _, bd = gen_matrix(1, V, synth.STREAM_THETA, 0.5, dtype)
        bd = bd.reshape(V)
    y = gen_labels(N, V, "zipf" if V > 1000 else "uniform", ign, noor)
    yd = torch.from_numpy(y).to(dev())
    out = bom.bom_head_forward_residual(Hd, Wd, yd, b=bd)
    Zref = bom.bom_head_forward(Hd, Wd, bd)
    torch.cuda.synchronize()
    Zg = out["Z"]
    zb = lambda t: t.view(torch.int16).cpu().numpy() if t.dtype == torch.bfloat16 else t.cpu().numpy().view(np.int32)
    assert np.array_equal(zb(Zg), zb(Zref)), f"{name}: Z differs from bom_head_forward"
    Zh = to_f64(Zg)
    o = oracle.residual(Zh, y)
    _compare_residual(name, Zh, y, out, o, dtype)
    ref = bom.bom_residual(Zg, yd)
    torch.cuda.synchronize()
    for k in ("row_argmax", "n_valid", "flags"):
        assert torch.equal(out[k], ref[k]), k
    assert torch.equal(out["row_target"], ref["row_target"])


def test_head_forward_residual_argmax_ties_across_tiles():
    # H = 0: every row of Z is the bias; its maximum sits at columns 700 and 5 (tiles 2 and 0) and twice in
    # tile 1: the first column (5) must win, as the oracle's lowest-index rule says
    N, d, V = 64, 64, 1024
    Hd = torch.zeros((N, d), dtype=torch.bfloat16, device=dev())
    Wd = torch.zeros((d, V), dtype=torch.bfloat16, device=dev())
    b = torch.full((V,), -1.0, dtype=torch.float32)
    b[[700, 5, 300, 301]] = 2.0
    bd = b.to(torch.bfloat16).to(dev())
    y = gen_labels(N, V, "uniform")
    out = bom.bom_head_forward_residual(Hd, Wd, torch.from_numpy(y).to(dev()), b=bd)
    torch.cuda.synchronize()
    assert (out["row_argmax"].cpu().numpy() == 5).all()
    Zh = to_f64(out["Z"])
    _compare_residual("ties", Zh, y, out, oracle.residual(Zh, y), "bf16")
