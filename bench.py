"""Benchmark of the BOM per-step hot path on one MI355X.

A step is one pass of the whole hot path over one synthetic batch resident in HBM:
  bom_residual (row statistics, R, s) -> bom_ema (q, q_hat) -> bom_head_vjp (dW into the head
  slice of the flat u, dH) -> bom_update (second moment and parameters over the flat buffer).
W untimed warmup steps, then exactly K timed steps bracketed by device synchronisation.
Per-stage durations come from HIP events recorded on the stream the kernels run on.

Prints one JSON line: whole-job tokens/s (rows of Z per second), per-stage times, the roofline
of the dominant stage, and the fp64 CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import re
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402
from synth.workloads import BY_NAME, WORKLOADS  # noqa: E402
from paper_2609_36738_amd import bom  # noqa: E402

HBM_PEAK_GBS = 8000.0      # MI355X HBM3E
MFMA_BF16_PEAK_TFS = 2500.0  # MI355X dense bf16 MFMA
FP32_PEAK_TFS = 157.3      # MI355X fp32 vector
METRIC = "BOM steps/s & tokens/s per config; % of HBM BW / MFMA peak per kernel"
# the headline: the largest workload that fits one GPU (the 8B-class language-model step); a default run
# also measures every other workload and reports it under "per_config"
HEADLINE_WORKLOAD = "lm_8b_v128256"
KERNEL_SOURCES = {
    "bom_residual": "residual.hip",
    "bom_ema": "ema.hip",
    "bom_head_vjp": "head_vjp.hip",
    "bom_update": "update.hip",
}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def source_hash(stage: str) -> str:
    path = os.path.join(ROOT, "paper_2609_36738_amd", "csrc", KERNEL_SOURCES[stage])
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def bf16_dev(bits: np.ndarray, shape, dev):
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).reshape(shape).to(dev)


def fill_normal_(t: torch.Tensor, stream: int, std: float, chunk: int = 1 << 27):
    """Fill a flat device tensor from the seeded generator (fp32 values, rounded to nearest-even on the copy
    into a bf16 tensor), chunk by chunk (bounded host memory)."""
    n = t.numel()
    host = np.empty(min(chunk, n), np.float32)
    for k, start in enumerate(range(0, n, chunk)):
        m = min(chunk, n - start)
        synth.normal_f32(m, stream, std, start=start, out=host[:m])
        t[start:start + m].copy_(torch.from_numpy(host[:m]))
        if k % 16 == 15:
            log(f"[bench] generated {start + m} of {n} values of stream {stream}")


def adam_mini_partition(w):
    """Segments tiling the flat buffer and their block lengths, shaped like Adam-mini's partition of a
    transformer: the head slice and the bias per element (the class blocks of Adam-mini's classifier branch
    are columns of the [d, V] head here, not contiguous), then the backbone with one sixth in per-head blocks
    (64 rows of d: query and key are 2 of a layer's 12 d x d matrices) and the rest per output neuron
    (blocks of d)."""
    hp = w.head_params
    segs, blocks = [(0, w.d * w.V, w.weight_decay)], [1]
    if w.has_bias:
        segs.append((w.d * w.V, w.V, 0.0))
        blocks.append(1)
    rest = w.P - hp
    blk_head = 64 * w.d
    n_head = (rest // 6) // blk_head * blk_head
    if n_head > 0:
        segs.append((hp, n_head, w.weight_decay))
        blocks.append(blk_head)
    if rest - n_head > 0:
        segs.append((hp + n_head, rest - n_head, w.weight_decay))
        blocks.append(w.d)
    return segs, blocks


class Problem:
    """Device-resident inputs and state of one workload."""

    def __init__(self, w, dev, clip_norm=0.0, state_dtype=torch.float32, adam_mini=False, z_route=False):
        self.w = w
        self.z_route = z_route
        self.blocks = None
        self.clip_norm = clip_norm
        self.state_dtype = state_dtype
        N, d, V, P = w.N, w.d, w.V, w.P
        std_z = w.logit_std
        t0 = time.time()
        if w.dtype == "bf16":
            self.Z = bf16_dev(synth.normal_bf16(N * V, synth.STREAM_Z, std_z), (N, V), dev)
            self.H = bf16_dev(synth.normal_bf16(N * d, synth.STREAM_H, 1.0), (N, d), dev)
            self.W = bf16_dev(synth.normal_bf16(d * V, synth.STREAM_W, 0.02), (d, V), dev)
        else:
            self.Z = torch.from_numpy(synth.normal_f32(N * V, synth.STREAM_Z, std_z).reshape(N, V)).to(dev)
            self.H = torch.from_numpy(synth.normal_f32(N * d, synth.STREAM_H, 1.0).reshape(N, d)).to(dev)
            self.W = None  # the tiny head reads W from theta
        y = synth.labels_uniform(N, V) if w.labels == "uniform" else synth.labels_zipf(N, V)
        self.labels = torch.from_numpy(y).to(dev)
        # the logits route forms R inside the head products: no R buffer
        self.R = None if z_route else torch.empty((N, V), dtype=self.Z.dtype, device=dev)
        self.theta = torch.empty(P, dtype=state_dtype, device=dev)
        fill_normal_(self.theta, synth.STREAM_THETA, 0.02)
        if w.dtype == "f32":
            self.theta[d * V:d * V + V].zero_()   # bias starts at 0
        self.u = torch.empty(P, dtype=state_dtype, device=dev)
        fill_normal_(self.u, synth.STREAM_U + 1, 1e-3)
        if adam_mini:
            self.segments, self.blocks = adam_mini_partition(w)
            self.v = torch.zeros(bom.blocks_count(self.segments, self.blocks), dtype=torch.float32, device=dev)
            self.v_col = None
        elif w.factored:
            nrows = -(-P // w.block_cols)
            nblocks = -(-nrows // w.block_rows)
            self.v = torch.zeros(nrows, dtype=torch.float32, device=dev)
            self.v_col = torch.zeros(nblocks * w.block_cols, dtype=torch.float32, device=dev)
        else:
            self.v = torch.zeros(P, dtype=state_dtype, device=dev)
            self.v_col = None
        self.q = torch.zeros(V, dtype=torch.float32, device=dev)
        self.q_hat = torch.empty(V, dtype=torch.float32, device=dev)
        self.dH = torch.empty((N, d), dtype=self.Z.dtype, device=dev)
        if not adam_mini:
            self.segments = w.segments()
        # outputs and workspaces allocated once
        self.res = None
        self.ws_res = self.ws_vjp = self.ws_upd = None
        torch.cuda.synchronize()
        log(f"[bench] inputs for {w.name} ready in {time.time() - t0:.1f}s")

    def init_adamw(self):
        """State of the comparison arm: AdamW's first moment m and its own second moment (dense, or the same
        factored layout as BOM's), on the same parameter and gradient buffers."""
        w = self.w
        dev = self.theta.device
        self.m = torch.zeros(w.P, dtype=torch.float32, device=dev)
        if w.factored:
            nrows = -(-w.P // w.block_cols)
            nblocks = -(-nrows // w.block_rows)
            self.va = torch.zeros(nrows, dtype=torch.float32, device=dev)
            self.va_col = torch.zeros(nblocks * w.block_cols, dtype=torch.float32, device=dev)
        else:
            self.va = torch.zeros(w.P, dtype=torch.float32, device=dev)
            self.va_col = None
        self.ws_adamw = None
        torch.cuda.synchronize()

    def step_adamw(self, t: int, ev=None):
        """One step of the AdamW arm: the same residual (the cross-entropy backward needs R), the head
        products at lambda = 0 (the plain gradient, no history term) and AdamW's update with its first
        moment. Stage events: residual, (no EMA), head VJP, update."""
        w = self.w
        d, V = w.d, w.V
        if ev is not None:
            ev[0].record()
        self.res = bom.bom_residual(self.Z, self.labels, R=self.R, workspace=self.ws_res,
                                    **({} if self.res is None else {k: self.res[k] for k in (
                                        "s", "row_lse", "row_argmax", "row_target", "loss", "n_valid", "flags")}))
        self.ws_res = self.res["workspace"]
        if ev is not None:
            ev[1].record()
            ev[2].record()
        W = self.W if self.W is not None else self.theta[: d * V].view(d, V)
        dW = self.u[: d * V].view(d, V)
        db = self.u[d * V: d * V + V] if w.has_bias else None
        g = bom.bom_head_vjp(self.H, W, self.R, self.labels, self.q_hat, self.res["n_valid"], s=self.res["s"],
                             lam=0.0, dW=dW, db=db, dH=self.dH, workspace=self.ws_vjp)
        self.ws_vjp = g["workspace"]
        if ev is not None:
            ev[3].record()
        cfg = bom.make_update_cfg(lr=w.lr, beta2=w.beta2, eps=w.eps, t=t, factored=w.factored,
                                  block_rows=w.block_rows, block_cols=w.block_cols)
        self.ws_adamw = bom.bom_adamw_update(self.theta, self.m, self.va, self.u, cfg, beta1=w.beta1,
                                             v_col=self.va_col, segments=self.segments, workspace=self.ws_adamw)
        if ev is not None:
            ev[4].record()

    def step(self, t: int, ev=None):
        w = self.w
        d, V = w.d, w.V
        if ev is not None:
            ev[0].record()
        self.res = bom.bom_residual(self.Z, self.labels, R=self.R, write_R=not self.z_route, workspace=self.ws_res,
                                    **({} if self.res is None else {k: self.res[k] for k in (
                                        "s", "row_lse", "row_argmax", "row_target", "loss", "n_valid", "flags")}))
        self.ws_res = self.res["workspace"]
        if ev is not None:
            ev[1].record()
        bom.bom_ema(self.q, self.res["s"], w.beta1, t, q_hat=self.q_hat)
        if ev is not None:
            ev[2].record()
        W = self.W if self.W is not None else self.theta[: d * V].view(d, V)
        dW = self.u[: d * V].view(d, V)
        db = self.u[d * V: d * V + V] if w.has_bias else None
        if self.z_route:
            g = bom.bom_head_vjp(self.H, W, self.Z, self.labels, self.q_hat, self.res["n_valid"], s=self.res["s"],
                                 lam=w.lam, dW=dW, db=db, dH=self.dH, workspace=self.ws_vjp,
                                 row_lse=self.res["row_lse"])
        else:
            g = bom.bom_head_vjp(self.H, W, self.R, self.labels, self.q_hat, self.res["n_valid"], s=self.res["s"],
                                 lam=w.lam, dW=dW, db=db, dH=self.dH, workspace=self.ws_vjp)
        self.ws_vjp = g["workspace"]
        if ev is not None:
            ev[3].record()
        cfg = bom.make_update_cfg(lr=w.lr, beta2=w.beta2, eps=w.eps, t=t, lam=w.lam,
                                  factored=w.factored and self.blocks is None, block_rows=w.block_rows,
                                  block_cols=w.block_cols, clip_norm=self.clip_norm, state_dtype=self.state_dtype,
                                  blocks=self.blocks)
        self.ws_upd = bom.bom_update(self.theta, self.v, self.u, cfg, v_col=self.v_col, segments=self.segments,
                                     workspace=self.ws_upd)
        if ev is not None:
            ev[4].record()


def time_graph(prob, args, t):
    """One step captured in a HIP graph (the library's launches on torch's capture stream) and replayed
    `steps` times: the step without the host's launch overhead (a replay repeats the captured step counter,
    whose bias corrections are kernel arguments, so this times the same work, not the same trajectory)."""
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        prob.step(t + 1)
    for _ in range(3):
        g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    del g
    log(f"[bench] {prob.w.name}: graph replay {ms:.4f} ms/step")
    return {"ms_per_step": round(ms, 5), "us_per_step": round(ms * 1e3, 2),
            "value": round(int(prob.res["n_valid"].item()) / (ms / 1e3), 1), "unit": "tokens/s"}


def time_adamw_arm(prob, args, bom_ms):
    """The AdamW arm on the same inputs (W warmup and K timed steps, like the BOM arm): step time, stage
    times, its update against the HBM roofline (28 bytes per parameter dense: read theta, m, v, g; write
    theta, m, v; factored second moment: 24 bytes, g read twice), and Delta t = t_BOM - t_AdamW."""
    w = prob.w
    prob.init_adamw()
    for k in range(args.warmup):
        prob.step_adamw(k + 1)
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for k in range(args.steps):
        prob.step_adamw(args.warmup + k + 1, evs[k])
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / args.steps
    st = {name: float(np.mean([evs[k][i].elapsed_time(evs[k][i + 1]) for k in range(args.steps)]))
          for i, name in ((0, "residual"), (2, "head_vjp"), (3, "update"))}
    nbytes = (24 if w.factored else 28) * w.P + (8 * -(-w.P // w.block_cols) if w.factored else 0)
    rate = nbytes / (st["update"] / 1e3) / 1e9
    del prob.m, prob.va, prob.va_col
    torch.cuda.empty_cache()
    log(f"[bench] {w.name}: AdamW arm {ms:.4f} ms/step (BOM {bom_ms:.4f})")
    return {"ms_per_step": round(ms, 5), "stages_ms": {k: round(v, 5) for k, v in st.items()},
            "bom_stages_ms": None,   # filled by run_workload
            "update": {"rate": round(rate, 2), "unit": "GB/s", "frac": round(rate / HBM_PEAK_GBS, 4),
                       "algorithmic_bytes": nbytes,
                       "per_unit": "24 bytes per parameter (factored v: read g twice, read+write theta and m)"
                       if w.factored else "28 bytes per parameter (read theta, m, v, g; write theta, m, v)"},
            "delta_ms": round(bom_ms - ms, 5), "ratio": round(bom_ms / ms, 5),
            "N_out": w.N * w.V, "P": w.P}


def cost_model_fit(rows):
    """Delta t = t_BOM - t_AdamW = alpha N_out - beta P (appendix 'First-order cost accounting'), alpha and beta
    in ms per 1e9 elements, r* = alpha / beta. 'joint': the paper's rule, least squares without intercept of
    the step-time differences on (N_out, -P). 'by_stage': each term on its own stages (the residual is the
    same call in both arms): the output side, EMA + head VJP (BOM) - head VJP (AdamW, lambda = 0), regressed
    on N_out; the parameter side, update (AdamW) - update (BOM), regressed on P. Across these workloads N_out
    and P grow together, so the joint fit is poorly conditioned and the staged one separates the terms."""
    A = np.array([[r["N_out"] / 1e9, -r["P"] / 1e9] for r in rows])
    y = np.array([r["delta_ms"] for r in rows])
    (alpha, beta), *_ = np.linalg.lstsq(A, y, rcond=None)
    pred = A @ np.array([alpha, beta])
    n_out = np.array([r["N_out"] / 1e9 for r in rows])
    p_par = np.array([r["P"] / 1e9 for r in rows])
    d_out = np.array([r["bom_stages_ms"]["bom_ema"] + r["bom_stages_ms"]["bom_head_vjp"] - r["stages_ms"]["head_vjp"]
                      for r in rows])
    d_par = np.array([r["stages_ms"]["update"] - r["bom_stages_ms"]["bom_update"] for r in rows])
    a_s = float(n_out @ d_out / (n_out @ n_out))
    b_s = float(p_par @ d_par / (p_par @ p_par))
    return {"joint": {"alpha_ms_per_1e9_nout": round(float(alpha), 4), "beta_ms_per_1e9_params": round(float(beta), 4),
                      "r_star": round(float(alpha / beta), 4) if beta != 0 else None},
            "by_stage": {"alpha_ms_per_1e9_nout": round(a_s, 4), "beta_ms_per_1e9_params": round(b_s, 4),
                         "r_star": round(a_s / b_s, 4) if b_s != 0 else None},
            "points": [{"workload": r["workload"], "N_out": r["N_out"], "P": r["P"], "delta_ms": r["delta_ms"],
                        "joint_fit_ms": round(float(p_), 4), "output_side_ms": round(float(do), 5),
                        "parameter_side_ms": round(float(dp), 5)}
                       for r, p_, do, dp in zip(rows, pred, d_out, d_par)],
            "paper_h800_context": {"alpha_ms_per_1e9_nout": 43.2758, "beta_ms_per_1e9_params": 15.4769,
                                   "r_star": 2.80}}


def time_forward(prob, steps):
    """Mean time of the head forward Z = H W (+ b) over `steps` calls into a scratch Z, and its rate
    against the bf16 MFMA peak (fp32 vector peak for the fp32 tiny head): 2 N d V flop."""
    w = prob.w
    W = prob.W if prob.W is not None else prob.theta[: w.d * w.V].view(w.d, w.V)
    b = None if not w.has_bias else prob.theta[w.d * w.V: w.d * w.V + w.V]
    Z = torch.empty_like(prob.Z)
    for _ in range(3):
        bom.bom_head_forward(prob.H, W, b, Z=Z)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        bom.bom_head_forward(prob.H, W, b, Z=Z)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    tf = 2.0 * w.N * w.d * w.V / (ms / 1e3) / 1e12
    peak = MFMA_BF16_PEAK_TFS if w.dtype == "bf16" else FP32_PEAK_TFS
    del Z
    return {"ms": round(ms, 5), "rate": round(tf, 2), "unit": "TFLOP/s", "frac": round(tf / peak, 4),
            "algorithmic_flop": 2 * w.N * w.d * w.V}


def time_forward_residual(prob, steps):
    """The head forward followed by the residual, as two calls (bom_head_forward, bom_residual) and as the
    fused call (bom_head_forward_residual: row statistics from the forward's epilogue, then one pass over Z
    for R and s), each timed over `steps` calls into scratch Z and R; inputs H, W, labels of the workload."""
    w = prob.w
    W = prob.W if prob.W is not None else prob.theta[: w.d * w.V].view(w.d, w.V)
    b = None if not w.has_bias else prob.theta[w.d * w.V: w.d * w.V + w.V]
    Z = torch.empty_like(prob.Z)
    R = torch.empty_like(prob.Z)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    res, ws = None, None

    def separate():
        nonlocal res, ws
        bom.bom_head_forward(prob.H, W, b, Z=Z)
        res = bom.bom_residual(Z, prob.labels, R=R, workspace=ws,
                               **({} if res is None else {k: res[k] for k in (
                                   "s", "row_lse", "row_argmax", "row_target", "loss", "n_valid", "flags")}))
        ws = res["workspace"]

    out, wsf = None, None

    def fused():
        nonlocal out, wsf
        out = bom.bom_head_forward_residual(prob.H, W, prob.labels, b=b, Z=Z, R=R, out=out, workspace=wsf)
        wsf = out["workspace"]

    times = {}
    for name, fn in (("separate", separate), ("fused", fused)):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        times[name] = e0.elapsed_time(e1) / steps
    del Z, R, ws, wsf, res, out
    torch.cuda.empty_cache()
    return {"separate_ms": round(times["separate"], 5), "fused_ms": round(times["fused"], 5),
            "saved_ms": round(times["separate"] - times["fused"], 5)}


def time_telemetry(prob, steps):
    """Mean time of the drift telemetry call over `steps` calls (M_W, M_b updated each call), and its
    HBM rate against the algorithmic bytes: read R and H, read and write M_W (and M_b)."""
    w = prob.w
    d, V, N = w.d, w.V, w.N
    esz = 2 if w.dtype == "bf16" else 4
    MW = torch.zeros((d, V), dtype=torch.float32, device=prob.Z.device)
    Mb = torch.zeros(V, dtype=torch.float32, device=prob.Z.device) if w.has_bias else None
    res = prob.res
    ws = None
    for k in range(3):
        ws = bom.bom_head_telemetry(prob.H, prob.R, prob.labels, res["s"], prob.q_hat, res["n_valid"], MW, M_b=Mb,
                                    beta1=w.beta1, t=k + 1, workspace=ws)["workspace"]
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for k in range(steps):
        tel = bom.bom_head_telemetry(prob.H, prob.R, prob.labels, res["s"], prob.q_hat, res["n_valid"], MW, M_b=Mb,
                                     beta1=w.beta1, t=k + 4, workspace=ws)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    nbytes = N * V * esz + N * d * esz + 8 * d * V + (8 * V if w.has_bias else 0)
    stats = dict(zip(bom.TELEMETRY_FIELDS, [round(float(x), 6) for x in tel["out"].cpu()]))
    return {"ms": round(ms, 5), "rate": round(nbytes / (ms / 1e3) / 1e9, 2), "unit": "GB/s",
            "frac": round(nbytes / (ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4), "algorithmic_bytes": nbytes,
            "last": stats}


def algorithmic(w, clip=False, bf16_state=False, blocks=None, z_route=False):
    """Algorithmic bytes / flops of each stage for one step (what BOM must move or compute). With
    global-norm clipping the dense update reads u once more for the norm; the factored update takes
    the norm from its row statistics (a row-sized array written once and read twice). blocks: the
    (segments, block lengths) of the block-shared second moment. z_route: the residual writes no R (the
    head products form it from Z)."""
    esz = 2 if w.dtype == "bf16" else 4
    N, d, V, P = w.N, w.d, w.V, w.P
    out = {
        "bom_residual": (dict(bound="hbm", amount=N * V * esz + 16 * N + 4 * V,
                              per_unit="esz bytes per logit (read Z) + 16 B/row + 4 B/column") if z_route else
                         dict(bound="hbm", amount=2 * N * V * esz + 16 * N + 4 * V,
                              per_unit="2*esz bytes per logit (read Z, write R) + 16 B/row + 4 B/column")),
        "bom_ema": dict(bound="hbm", amount=12 * V, per_unit="12 bytes per output coordinate"),
        "bom_head_vjp": dict(bound="mfma" if w.dtype == "bf16" else "alu", amount=4 * N * d * V,
                             per_unit="4*N*d*V flop (dW and dH)"),
    }
    if blocks is not None:
        # per element: 20 B (read theta, v, u; write theta, v); blocks of up to 4096: 12 B (read u, theta;
        # write theta); longer blocks: 16 B (u read twice); 8 B per block entry of v; clipping: 4 B more
        amount = 0
        for (o, n, _), bk in zip(*blocks):
            per = 20 if bk == 1 else (12 if min(bk, n) <= 4096 else 16)
            amount += per * n + (0 if bk == 1 else 8 * -(-n // bk)) + (4 * n if clip else 0)
        out["bom_update"] = dict(bound="hbm", amount=amount,
                                 per_unit="20 B per parameter with its own v, 12 B in blocks of up to 4096 (read u "
                                          "and theta, write theta), 16 B in longer blocks (u read twice), 8 B per "
                                          "block" + ("; +4 B per parameter for the norm" if clip else ""))
    elif w.factored:
        nrows = -(-P // w.block_cols)
        nblocks = -(-nrows // w.block_rows)
        out["bom_update"] = dict(bound="hbm", amount=16 * P + 8 * nrows + 8 * nblocks * w.block_cols
                                 + (12 * nrows if clip else 0),
                                 per_unit="16 bytes per parameter (read u twice, read+write theta) + factors")
    elif bf16_state:
        out["bom_update"] = dict(bound="hbm", amount=(12 if clip else 10) * P,
                                 per_unit=f"{12 if clip else 10} bytes per parameter (bf16 storage: "
                                          f"{'read u for the norm; ' if clip else ''}read theta, v, u; write theta, v)")
    elif clip:
        out["bom_update"] = dict(bound="hbm", amount=24 * P, per_unit="24 bytes per parameter (read u for the norm; "
                                                                      "read theta, v, u; write theta, v)")
    else:
        out["bom_update"] = dict(bound="hbm", amount=20 * P, per_unit="20 bytes per parameter (read theta, v, u; "
                                                                      "write theta, v)")
    return out


def stored_traffic(stage: str, workload: str):
    """HBM traffic of a stage from a committed rocprofv3 counter summary, if the kernel source is unchanged."""
    path = os.path.join(ROOT, "profiles", f"{stage}_{workload}_counters.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_hash = re.search(r"source_sha256_16:\s*([0-9a-f]{16})", text)
    m_bytes = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m_hash or not m_bytes or m_hash.group(1) != source_hash(stage):
        return None
    return float(m_bytes.group(1))


def _oracle_sample(w, rows, ncols, nrows_dh, npar):
    """Host seconds of each oracle stage on one sample: `rows` rows of Z (residual; dW and dH use the
    same rows), `ncols` dW columns, `nrows_dh` dH rows, `npar` parameters of the update."""
    import oracle

    N, d, V = w.N, w.d, w.V
    raw = {}
    Zs = synth.bf16_to_f32(synth.normal_bf16(rows * V, synth.STREAM_Z, w.logit_std)) if w.dtype == "bf16" else \
        synth.normal_f32(rows * V, synth.STREAM_Z, w.logit_std)
    Zs = Zs.reshape(rows, V).astype(np.float64)
    y = (synth.labels_uniform(N, V) if w.labels == "uniform" else synth.labels_zipf(N, V))[:rows]
    t0 = time.perf_counter()
    res = oracle.residual(Zs, y, want_R=False)
    raw["bom_residual"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    _, qh = oracle.ema(np.zeros(V), res["s"], w.beta1, 1)
    raw["bom_ema"] = time.perf_counter() - t0
    Hs = synth.normal_f32(rows * d, synth.STREAM_H, 1.0).reshape(rows, d).astype(np.float64)
    Ws = synth.normal_f32(d * V, synth.STREAM_W, 0.02).reshape(d, V).astype(np.float64)
    t0 = time.perf_counter()
    oracle.dW_cols(Hs, Zs, y, res["row_lse"], qh, res["n_valid"], w.lam, cols=np.arange(ncols))
    raw["dW"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.dH_rows(Ws, Zs, y, res["row_lse"], qh, res["n_valid"], w.lam, rows=np.arange(nrows_dh))
    raw["dH"] = time.perf_counter() - t0
    del Zs, Hs, Ws
    th = synth.normal_f32(npar, synth.STREAM_THETA, 0.02).astype(np.float64)
    u = synth.normal_f32(npar, synth.STREAM_U + 1, 1e-3).astype(np.float64)
    t0 = time.perf_counter()
    if w.factored:
        bc, br = w.block_cols, w.block_rows
        nr = npar // bc
        oracle.update_factored(th[: nr * bc], np.zeros(nr), np.zeros(-(-nr // br) * bc), u[: nr * bc], lr=w.lr,
                               beta2=w.beta2, eps=w.eps, t=1, block_rows=br, block_cols=bc,
                               weight_decay=w.weight_decay)
        npar = nr * bc
    else:
        oracle.update_dense(th, np.zeros(npar), u, lr=w.lr, beta2=w.beta2, eps=w.eps, t=1,
                            weight_decay=w.weight_decay)
    raw["bom_update"] = time.perf_counter() - t0
    # each stage scaled linearly to the whole step
    full = {"bom_residual": raw["bom_residual"] * N / rows, "bom_ema": raw["bom_ema"],
            "bom_head_vjp": raw["dW"] * (V / ncols) * (N / rows) + raw["dH"] * (N / nrows_dh),
            "bom_update": raw["bom_update"] * w.P / npar}
    return raw, full, npar


def cpu_baseline(w, budget_s: float):
    """The fp64 oracle (as it stands) timed on the host on a bounded sample of the same workload,
    scaled to the whole step. Starting from a small probe, the sample of each part (residual rows,
    head-product columns and rows, update parameters) grows until that part takes about a third of
    `budget_s`, covers the whole workload or reaches its host-memory bound; the final sample is then
    repeated until two thirds of the budget is used, and the mean over the repetitions is reported."""
    N, d, V, P = w.N, w.d, w.V, w.P
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    max_rows = max(16, min(N, int(4e7 // V), int(4e7 // d)))     # bounded host memory (fp64 copies)
    max_par = min(P, 200_000_000)
    rows = min(max_rows, max(16, int(2e6 // V)))
    ncols, nrows_dh, npar = min(V, 64), min(rows, 16), min(max_par, 4_000_000)
    share = budget_s / 3.0
    spent = 0.0
    for _ in range(4):
        raw, full, npar = _oracle_sample(w, rows, ncols, nrows_dh, npar)
        spent += sum(raw.values())
        grown = False
        if raw["bom_residual"] < 0.5 * share and rows < max_rows:
            f = min(8.0, share / max(raw["bom_residual"], 1e-4))
            rows, grown = int(min(max_rows, rows * f)), True
        vjp = raw["dW"] + raw["dH"]
        if vjp < 0.5 * share and (ncols < V or nrows_dh < rows):
            f = min(8.0, share / max(vjp, 1e-4))
            ncols, nrows_dh, grown = int(min(V, ncols * f)), int(min(rows, nrows_dh * f)), True
        nrows_dh = min(nrows_dh, rows)
        if raw["bom_update"] < 0.5 * share and npar < max_par:
            f = min(8.0, share / max(raw["bom_update"], 1e-4))
            npar, grown = int(min(max_par, npar * f)), True
        if not grown:
            break
    else:
        raw, full, npar = _oracle_sample(w, rows, ncols, nrows_dh, npar)
        spent += sum(raw.values())
    whole = rows == N and ncols == V and nrows_dh == N and npar == P
    reps, t_sample, acc = 1, sum(raw.values()), dict(full)
    while t_sample < budget_s * 2.0 / 3.0 and reps < 200:
        raw, full, npar = _oracle_sample(w, rows, ncols, nrows_dh, npar)
        t_sample += sum(raw.values())
        reps += 1
        acc = {k: acc[k] + full[k] for k in full}
    t_all = {k: v / reps for k, v in acc.items()}
    step_s = sum(t_all.values())
    sample = ("the whole step (all rows, full dW and dH, all parameters)" if whole else
              f"{rows} of {N} rows of Z (residual; dW and dH on the same rows), {ncols} of {V} dW columns, "
              f"{nrows_dh} of {N} dH rows, {npar} of {P} parameters (update); each stage scaled linearly to "
              f"the full step")
    return {
        "value": N / step_s, "unit": "tokens/s", "cores": cores, "kind": "oracle",
        "sample": f"{sample}; {reps} repetition(s), {t_sample:.1f} s of oracle time",
        "step_s_extrapolated": step_s,
        "stage_s": {k: round(v, 4) for k, v in t_all.items()},
        "nproc": os.cpu_count(), "host_cpu": host_cpu_model(),
    }


def host_cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def run_workload(w, args, cpu_budget, dev):
    """Inputs of workload w resident in HBM, W warmup steps, K timed steps, per-stage times from HIP events,
    the roofline of the dominant stage and the oracle baseline. Returns the JSON object of this workload."""
    state_dtype = torch.bfloat16 if args.state_dtype == "bf16" else torch.float32
    prob = Problem(w, dev, clip_norm=args.clip_norm, state_dtype=state_dtype, adam_mini=args.adam_mini,
                   z_route=args.z_route)
    stages = ["bom_residual", "bom_ema", "bom_head_vjp", "bom_update"]

    t = 0
    for _ in range(args.warmup):
        t += 1
        prob.step(t)
    torch.cuda.synchronize()
    log(f"[bench] {w.name}: warmup {args.warmup} steps done")

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record()
    for k in range(args.steps):
        t += 1
        prob.step(t, evs[k])
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = start.elapsed_time(end)
    ms_per_step = total_ms / args.steps
    per_step = np.array([evs[k][0].elapsed_time(evs[k][4]) for k in range(args.steps)])
    stage_ms = {s: float(np.mean([evs[k][i].elapsed_time(evs[k][i + 1]) for k in range(args.steps)]))
                for i, s in enumerate(stages)}
    log(f"[bench] {w.name}: timed {args.steps} steps: {ms_per_step:.4f} ms/step (wall {wall:.2f}s)")

    alg = algorithmic(w, clip=args.clip_norm > 0, bf16_state=state_dtype == torch.bfloat16,
                      blocks=(prob.segments, prob.blocks) if args.adam_mini else None, z_route=args.z_route)
    dom = max(stages, key=lambda s: stage_ms[s])
    a = alg[dom]
    sec = stage_ms[dom] / 1e3
    if a["bound"] == "hbm":
        achieved, peak, unit = a["amount"] / sec / 1e9, HBM_PEAK_GBS, "GB/s"
    elif a["bound"] == "mfma":
        achieved, peak, unit = a["amount"] / sec / 1e12, MFMA_BF16_PEAK_TFS, "TFLOP/s"
    else:
        achieved, peak, unit = a["amount"] / sec / 1e12, FP32_PEAK_TFS, "TFLOP/s"
    roofline = {"bound": a["bound"], "achieved": round(achieved, 2), "peak": peak, "unit": unit,
                "frac": round(achieved / peak, 4),
                "traffic": (stored_traffic(dom, w.name)
                            if args.clip_norm == 0 and args.state_dtype == "f32" and not args.adam_mini
                            and not args.z_route else None),
                "kernel": dom,
                "algorithmic_per_launch": a["amount"], "per_unit": a["per_unit"]}
    per_stage = {}
    for s in stages:
        b = alg[s]
        ss = stage_ms[s] / 1e3
        rate = b["amount"] / ss / (1e9 if b["bound"] == "hbm" else 1e12)
        pk = HBM_PEAK_GBS if b["bound"] == "hbm" else (MFMA_BF16_PEAK_TFS if b["bound"] == "mfma" else FP32_PEAK_TFS)
        per_stage[s] = {"ms": round(stage_ms[s], 5), "us": round(stage_ms[s] * 1e3, 2), "rate": round(rate, 2),
                        "unit": "GB/s" if b["bound"] == "hbm" else "TFLOP/s", "frac": round(rate / pk, 4)}

    n_valid = int(prob.res["n_valid"].item())
    out = {
        "value": round(n_valid / (ms_per_step / 1e3), 1),
        "unit": "tokens/s",
        "ms_per_step": round(ms_per_step, 5),
        "us_per_step": round(ms_per_step * 1e3, 2),
        "steps_per_s": round(1e3 / ms_per_step, 2),
        "median_ms_per_step": round(float(np.median(per_step)), 5),
        "p10_p90_ms": [round(float(np.percentile(per_step, 10)), 5), round(float(np.percentile(per_step, 90)), 5)],
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "config": {"workload": w.name, "N": w.N, "d": w.d, "V": w.V, "P": w.P, "tokens_per_step": n_valid,
                   "second_moment": "blocks" if args.adam_mini else ("factored" if w.factored else "dense"),
                   "clip_norm": args.clip_norm,
                   "state_dtype": args.state_dtype,
                   "head_input": "logits" if args.z_route else "residual"},
        "stages": per_stage,
        "roofline": roofline,
    }
    if args.graph:
        out["graph"] = time_graph(prob, args, t)
    if args.adamw:
        out["adamw"] = time_adamw_arm(prob, args, ms_per_step)
        out["adamw"]["bom_stages_ms"] = {s: round(stage_ms[s], 5) for s in stages}
    if args.forward:
        out["forward"] = time_forward(prob, args.steps)
    if args.fused_forward:
        out["forward_residual"] = time_forward_residual(prob, args.steps)
    if args.telemetry:
        out["telemetry"] = time_telemetry(prob, args.steps)
    del prob
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        log(f"[bench] {w.name}: timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(w, cpu_budget)
    else:
        out["cpu_baseline"] = None
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default=None, choices=[w.name for w in WORKLOADS],
                    help="measure only this workload (default: the 8B-class step as the headline, every other "
                         "workload under per_config)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--state-dtype", choices=["f32", "bf16"], default="f32",
                    help="storage of theta, v and u (bf16: the paper's fine-tuning protocol; dense layout, bf16 "
                         "logits only)")
    ap.add_argument("--forward", action="store_true",
                    help="also time the head forward Z = H W that produces the logits (common work, outside the "
                         "step) against the MFMA roofline")
    ap.add_argument("--fused-forward", action="store_true",
                    help="also time the head forward plus the residual as two calls and as the fused call with the "
                         "row statistics from the forward's epilogue (common work plus the residual, outside the step)")
    ap.add_argument("--telemetry", action="store_true",
                    help="also time the head drift telemetry call (a diagnostic for telemetry steps, outside the "
                         "step) on the last step's residual, history and features")
    ap.add_argument("--clip-norm", type=float, default=0.0,
                    help="global-norm clipping of the update numerator at this norm (0: none; the paper's "
                         "language-model protocols clip at 1.0)")
    ap.add_argument("--adam-mini", action="store_true",
                    help="block-shared second moment (Adam-mini's update map with the BOM numerator) over a "
                         "transformer-shaped partition of the flat buffer, instead of the dense or factored one")
    ap.add_argument("--graph", action="store_true",
                    help="also time one step captured in a HIP graph and replayed (no host launch overhead)")
    ap.add_argument("--no-adamw", dest="adamw", action="store_false",
                    help="skip the AdamW comparison arm (and the cost-model fit) after each workload's BOM steps")
    ap.add_argument("--z-route", action="store_true",
                    help="the head products take the logits Z and row_lse and form R themselves; the residual "
                         "writes no R")
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="host seconds the oracle baseline aims to spend on the headline workload")
    ap.add_argument("--cpu-budget-other", type=float, default=5.0,
                    help="host seconds the oracle baseline aims to spend on each per_config workload")
    ap.add_argument("--calibrate-copy-mb", type=int, default=0,
                    help="run an untimed plain device-to-device copy of this many MiB first (a known-size "
                         "reference for hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: the BOM hot path is implemented and measured on a single MI355X; "
              "its sharding across GPUs is described, not implemented.", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    bom.load(build_if_missing=False)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.calibrate_copy_mb > 0:
        nbytes = args.calibrate_copy_mb << 20
        src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy of {nbytes} bytes done (3 launches)")
        del src, dst
        torch.cuda.empty_cache()
    state_dtype = torch.bfloat16 if args.state_dtype == "bf16" else torch.float32
    headline = BY_NAME[args.workload or HEADLINE_WORKLOAD]
    others = [] if args.workload else [w for w in WORKLOADS if w.name != headline.name]
    for w in [headline] + others:
        if state_dtype == torch.bfloat16 and (w.factored or w.dtype != "bf16"):
            print(f"bf16 state storage applies to the dense layout with bf16 logits ({w.name} has neither); "
                  "pick a workload with --workload", file=sys.stderr)
            sys.exit(2)
    if args.adam_mini and state_dtype == torch.bfloat16:
        print("the block-shared second moment keeps fp32 state", file=sys.stderr)
        sys.exit(2)

    main_res = run_workload(headline, args, args.cpu_budget, dev)
    out = {
        "metric": METRIC,
        "value": main_res.pop("value"),
        "unit": main_res.pop("unit"),
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": main_res.pop("ms_per_step"),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": main_res.pop("dtype"),
        "data": "synthetic",
    }
    out.update(main_res)
    if others:
        out["per_config"] = {}
        for w in others:
            out["per_config"][w.name] = run_workload(w, args, args.cpu_budget_other, dev)
    if args.adamw:
        # the paper's ladder is the language-model pretraining rungs: fit over the bf16-logit workloads (the
        # tiny fp32 classifier is launch-bound, its Delta t a few microseconds of launch jitter)
        rows = [dict(r["adamw"], workload=r["config"]["workload"])
                for r in [out] + list(out.get("per_config", {}).values())
                if "adamw" in r and BY_NAME[r["config"]["workload"]].dtype == "bf16"]
        if len(rows) >= 2:
            out["cost_model"] = cost_model_fit(rows)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
