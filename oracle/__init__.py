"""fp64 CPU oracle for the BOM per-step hot path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's ``cpu_baseline`` leg may
import this package. It shares no code with the GPU library (``paper_2609_36738_amd``) and
never imports it. The arithmetic lives in ``bom_oracle.c`` (plain loops, fp64); this module
builds it with gcc, marshals numpy arrays, and strings the steps of Algorithm 1 together in
the paper's order for the multi-step loop.

Every function takes the exact fp64 images of the inputs (bf16 and fp32 widen exactly).
Pins: every function here is checked by ``tests/test_oracle_pins.py`` against what the paper
and the mathematics fix (closed forms, brute-force Jacobians, finite differences, explicit
EMA sums, Lemma 2, the linear-model equivalence of BOM and the own-step control, the
Adafactor rank-1 identity for the factored second moment, whose definition is a reading, and the
reduction of the block-shared second moment to the dense one at block length 1).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "bom_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

FLAG_LABEL_RANGE = 1
FLAG_EMPTY = 2


def build() -> str:
    cmd = ["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11", "-o", _LIB_PATH + ".tmp", _SRC, "-lm"]
    subprocess.check_call(cmd)
    os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        i64, i32, f64, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_double, ctypes.c_void_p
        lib.orc_residual.argtypes = [vp, i64, i64, vp, i32, vp, vp, vp, vp, vp, vp, vp, vp]
        lib.orc_ema.argtypes = [vp, vp, i64, f64, i64, vp]
        lib.orc_dW_cols.argtypes = [vp, i64, i64, vp, i64, vp, i32, vp, vp, i64, f64, vp, i64, vp]
        lib.orc_dH_rows.argtypes = [vp, i64, vp, i64, vp, i32, vp, vp, i64, f64, vp, i64, vp]
        lib.orc_dW_cols_sub.argtypes = [vp, i64, i64, vp, i64, vp, i32, vp, vp, i64, f64, vp, i64, vp]
        lib.orc_dH_rows_sub.argtypes = [vp, i64, vp, i64, vp, i32, vp, vp, i64, f64, vp, i64, vp]
        lib.orc_db.argtypes = [vp, i64, i64, vp, i32, vp, vp, i64, f64, vp]
        lib.orc_update_dense.argtypes = [vp, vp, vp, vp, i64, vp, vp, vp, ctypes.c_int, f64, f64, f64, f64, f64,
                                         f64, i64]
        lib.orc_update_factored.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, vp, vp, vp, ctypes.c_int, f64, f64,
                                            f64, f64, f64, f64, i64]
        lib.orc_update_blocks.argtypes = [vp, vp, vp, vp, i64, vp, vp, vp, vp, ctypes.c_int, f64, f64, f64, f64, f64,
                                          i64]
        lib.orc_update_adamw.argtypes = [vp, vp, vp, vp, i64, vp, vp, vp, ctypes.c_int, f64, f64, f64, f64, f64, f64,
                                         i64]
        lib.orc_update_adamw_factored.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, vp, vp, vp, ctypes.c_int, f64,
                                                  f64, f64, f64, f64, f64, i64]
        lib.orc_head_forward.argtypes = [vp, i64, i64, vp, i64, vp, vp]
        lib.orc_clip_factor.argtypes = [vp, vp, i64, f64, f64, f64]
        lib.orc_round_bf16.argtypes = [vp, i64, vp]
        lib.orc_head_telemetry.argtypes = [vp, i64, i64, vp, i64, vp, i32, vp, vp, i64, vp, vp, f64, i64, vp]
        lib.orc_clip_factor.restype = f64
        _lib = lib
        return lib


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def _p(a):
    return None if a is None else a.ctypes.data


def residual(Z, labels, ignore_index: int = -100, want_R: bool = True) -> dict:
    """Row statistics, residual rows, batch-mean residual s, mean CE, N_t and flags."""
    Z = _f64(Z)
    labels = _i32(labels)
    N, V = Z.shape
    out = dict(s=np.zeros(V), row_lse=np.zeros(N), row_argmax=np.zeros(N, np.int32),
               row_target=np.zeros(N), R=np.zeros((N, V)) if want_R else None)
    loss = np.zeros(1)
    nv = np.zeros(1, np.int32)
    fl = np.zeros(1, np.int32)
    _load().orc_residual(_p(Z), N, V, _p(labels), ignore_index, _p(out["s"]), _p(out["row_lse"]),
                         _p(out["row_argmax"]), _p(out["row_target"]), _p(out["R"]), _p(loss), _p(nv), _p(fl))
    out.update(loss=float(loss[0]), n_valid=int(nv[0]), flags=int(fl[0]))
    return out


def ema(q, s, beta1: float, t: int):
    """Returns (q_new, q_hat); the input q is not modified."""
    q = _f64(q).copy()
    s = _f64(s)
    qh = np.zeros_like(q)
    _load().orc_ema(_p(q), _p(s), q.size, float(beta1), int(t), _p(qh))
    return q, qh


def dW_cols(H, Z, labels, row_lse, q_hat, n_valid: int, lam: float, cols=None, ignore_index: int = -100):
    H, Z, labels, row_lse, q_hat = _f64(H), _f64(Z), _i32(labels), _f64(row_lse), _f64(q_hat)
    N, d = H.shape
    V = Z.shape[1]
    cols = np.arange(V, dtype=np.int64) if cols is None else np.ascontiguousarray(cols, dtype=np.int64)
    out = np.zeros((d, cols.size))
    _load().orc_dW_cols(_p(H), N, d, _p(Z), V, _p(labels), ignore_index, _p(row_lse), _p(q_hat), n_valid,
                        float(lam), _p(cols), cols.size, _p(out))
    return out


def dH_rows(W, Z, labels, row_lse, q_hat, n_valid: int, lam: float, rows=None, ignore_index: int = -100):
    W, Z, labels, row_lse, q_hat = _f64(W), _f64(Z), _i32(labels), _f64(row_lse), _f64(q_hat)
    d, V = W.shape
    N = Z.shape[0]
    rows = np.arange(N, dtype=np.int64) if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    out = np.zeros((rows.size, d))
    _load().orc_dH_rows(_p(W), d, _p(Z), V, _p(labels), ignore_index, _p(row_lse), _p(q_hat), n_valid,
                        float(lam), _p(rows), rows.size, _p(out))
    return out


def dW_cols_sub(H, Zcols, cols, V: int, labels, row_lse, q_hat, n_valid: int, lam: float, ignore_index: int = -100):
    """dW columns `cols` from the matching columns of Z only (Zcols is N x len(cols))."""
    H, Zc, labels, row_lse, q_hat = _f64(H), _f64(Zcols), _i32(labels), _f64(row_lse), _f64(q_hat)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    N, d = H.shape
    assert Zc.shape == (N, cols.size)
    out = np.zeros((d, cols.size))
    _load().orc_dW_cols_sub(_p(H), N, d, _p(Zc), V, _p(labels), ignore_index, _p(row_lse), _p(q_hat), n_valid,
                            float(lam), _p(cols), cols.size, _p(out))
    return out


def dH_rows_sub(W, Zrows, rows, labels, row_lse, q_hat, n_valid: int, lam: float, ignore_index: int = -100):
    """dH rows `rows` from the matching rows of Z only (Zrows is len(rows) x V); labels and row_lse
    are indexed by the full row numbers."""
    W, Zr, labels, row_lse, q_hat = _f64(W), _f64(Zrows), _i32(labels), _f64(row_lse), _f64(q_hat)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    d, V = W.shape
    assert Zr.shape == (rows.size, V)
    out = np.zeros((rows.size, d))
    _load().orc_dH_rows_sub(_p(W), d, _p(Zr), V, _p(labels), ignore_index, _p(row_lse), _p(q_hat), n_valid,
                            float(lam), _p(rows), rows.size, _p(out))
    return out


def db(Z, labels, row_lse, q_hat, n_valid: int, lam: float, ignore_index: int = -100):
    Z, labels, row_lse, q_hat = _f64(Z), _i32(labels), _f64(row_lse), _f64(q_hat)
    N, V = Z.shape
    out = np.zeros(V)
    _load().orc_db(_p(Z), N, V, _p(labels), ignore_index, _p(row_lse), _p(q_hat), n_valid, float(lam), _p(out))
    return out


def _segs(segments):
    segments = list(segments or [])
    off = np.array([s[0] for s in segments] or [0], np.int64)
    ln = np.array([s[1] for s in segments] or [0], np.int64)
    wd = np.array([s[2] for s in segments] or [0.0], np.float64)
    return off, ln, wd, len(segments)


def clip_factor(u, *, h=None, lam=0.5, u_scale=1.0, clip_norm=0.0) -> float:
    """Global-norm clipping factor of the update numerator: min(1, clip_norm / (||u'|| + 1e-6)); 1 when
    clip_norm <= 0 (no clipping)."""
    if clip_norm <= 0:
        return 1.0
    u = _f64(u)
    h = None if h is None else _f64(h)
    return float(_load().orc_clip_factor(_p(u), _p(h), u.size, float(lam), float(u_scale), float(clip_norm)))


def update_dense(theta, v, u, *, lr, beta2, eps, t, segments=None, weight_decay=0.0, h=None, lam=0.5,
                 u_scale=1.0, clip_norm=0.0):
    """Returns (theta_new, v_new) in fp64; inputs are not modified. clip_norm > 0 scales the numerator
    by clip_factor (global-norm clipping) before the second moment and the step."""
    theta, v, u = _f64(theta).copy(), _f64(v).copy(), _f64(u)
    h = None if h is None else _f64(h)
    u_scale = u_scale * clip_factor(u, h=h, lam=lam, u_scale=u_scale, clip_norm=clip_norm)
    off, ln, wd, ns = _segs(segments)
    _load().orc_update_dense(_p(theta), _p(v), _p(u), _p(h), theta.size, _p(off), _p(ln), _p(wd), ns,
                             float(weight_decay), float(lr), float(beta2), float(eps), float(lam), float(u_scale),
                             int(t))
    return theta, v


def update_adamw(theta, m, v, g, *, lr, beta1, beta2, eps, t, segments=None, weight_decay=0.0, u_scale=1.0):
    """AdamW step (the comparison arm of the cost model): returns (theta_new, m_new, v_new) in fp64."""
    theta, m, v, g = _f64(theta).copy(), _f64(m).copy(), _f64(v).copy(), _f64(g)
    off, ln, wd, ns = _segs(segments)
    _load().orc_update_adamw(_p(theta), _p(m), _p(v), _p(g), theta.size, _p(off), _p(ln), _p(wd), ns,
                             float(weight_decay), float(lr), float(beta1), float(beta2), float(eps), float(u_scale),
                             int(t))
    return theta, m, v


def update_adamw_factored(theta, m, Rr, Cc, g, *, lr, beta1, beta2, eps, t, block_rows, block_cols, segments=None,
                          weight_decay=0.0, u_scale=1.0):
    """AdamW with the factored second moment: returns (theta_new, m_new, Rr_new, Cc_new) in fp64."""
    theta, m, Rr, Cc, g = _f64(theta).copy(), _f64(m).copy(), _f64(Rr).copy(), _f64(Cc).copy(), _f64(g)
    off, ln, wd, ns = _segs(segments)
    _load().orc_update_adamw_factored(_p(theta), _p(m), _p(Rr), _p(Cc), _p(g), theta.size, int(block_rows),
                                      int(block_cols), _p(off), _p(ln), _p(wd), ns, float(weight_decay), float(lr),
                                      float(beta1), float(beta2), float(eps), float(u_scale), int(t))
    return theta, m, Rr, Cc


TELEMETRY_FIELDS = ("cos", "drift", "cancellation", "m_norm", "h_norm")


def head_telemetry(H, R, labels, s, q_hat, n_valid: int, M_W, M_b=None, *, beta1, t, ignore_index: int = -100):
    """One drift-telemetry step of the linear head. Returns (M_W_new, M_b_new or None, dict of
    TELEMETRY_FIELDS); inputs are not modified."""
    H, R, labels = _f64(H), _f64(R), _i32(labels)
    s, q_hat = _f64(s), _f64(q_hat)
    M_W = _f64(M_W).copy()
    M_b = None if M_b is None else _f64(M_b).copy()
    N, d = H.shape
    V = R.shape[1]
    out = np.zeros(5)
    _load().orc_head_telemetry(_p(H), N, d, _p(R), V, _p(labels), ignore_index, _p(s), _p(q_hat), int(n_valid),
                               _p(M_W), _p(M_b), float(beta1), int(t), _p(out))
    return M_W, M_b, dict(zip(TELEMETRY_FIELDS, out.tolist()))


def round_bf16(x) -> np.ndarray:
    """Bit patterns (uint16) of x rounded once from fp64 to the nearest bf16, ties to even."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty(x.shape, np.uint16)
    _load().orc_round_bf16(_p(x), x.size, out.ctypes.data_as(ctypes.c_void_p))
    return out


def bf16_bits_to_f64(bits) -> np.ndarray:
    """Exact fp64 images of bf16 bit patterns."""
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def update_dense_bf16(theta_bits, v_bits, u_bits, *, h_bits=None, **kw):
    """bf16 storage: the fp64 step (update_dense, same keywords) on the exact images of the bf16
    inputs, then theta and v rounded once to bf16. Returns their bit patterns."""
    th, v = update_dense(bf16_bits_to_f64(theta_bits), bf16_bits_to_f64(v_bits), bf16_bits_to_f64(u_bits),
                         h=None if h_bits is None else bf16_bits_to_f64(h_bits), **kw)
    return round_bf16(th), round_bf16(v)


def update_factored(theta, Rr, Cc, u, *, lr, beta2, eps, t, block_rows, block_cols, segments=None,
                    weight_decay=0.0, h=None, lam=0.5, u_scale=1.0, clip_norm=0.0):
    """Returns (theta_new, Rr_new, Cc_new) in fp64; inputs are not modified. clip_norm as in
    update_dense."""
    theta, Rr, Cc, u = _f64(theta).copy(), _f64(Rr).copy(), _f64(Cc).copy(), _f64(u)
    h = None if h is None else _f64(h)
    u_scale = u_scale * clip_factor(u, h=h, lam=lam, u_scale=u_scale, clip_norm=clip_norm)
    P = theta.size
    nrows = -(-P // block_cols)
    nblocks = -(-nrows // block_rows)
    assert Rr.size == nrows and Cc.size == nblocks * block_cols, "factored state shape"
    off, ln, wd, ns = _segs(segments)
    _load().orc_update_factored(_p(theta), _p(Rr), _p(Cc), _p(u), _p(h), P, block_rows, block_cols, _p(off), _p(ln),
                                _p(wd), ns, float(weight_decay), float(lr), float(beta2), float(eps), float(lam),
                                float(u_scale), int(t))
    return theta, Rr, Cc


def blocks_count(segments, blocks) -> int:
    """Entries of the block-shared second moment: sum over segments of ceil(length / block)."""
    return int(sum(-(-int(sg[1]) // int(bk)) for sg, bk in zip(segments, blocks)))


def update_blocks(theta, v, u, *, lr, beta2, eps, t, segments, blocks, h=None, lam=0.5, u_scale=1.0,
                  clip_norm=0.0):
    """Block-shared second moment (Adam-mini's map with the BOM numerator). segments = [(offset, length,
    weight_decay)] tiling [0, P) in order, blocks = block length per segment. Returns (theta_new, v_new)
    in fp64; inputs are not modified. clip_norm as in update_dense."""
    theta, v, u = _f64(theta).copy(), _f64(v).copy(), _f64(u)
    h = None if h is None else _f64(h)
    segments, blocks = list(segments), [int(b) for b in blocks]
    assert len(segments) == len(blocks) and segments, "one block length per segment"
    pos = 0
    for (o, n, _), bk in zip(segments, blocks):
        assert o == pos and n >= 1 and bk >= 1, "segments must tile [0, P) in order"
        pos += n
    assert pos == theta.size and v.size == blocks_count(segments, blocks), "block state shape"
    u_scale = u_scale * clip_factor(u, h=h, lam=lam, u_scale=u_scale, clip_norm=clip_norm)
    off, ln, wd, ns = _segs(segments)
    blk = np.array(blocks, np.int64)
    _load().orc_update_blocks(_p(theta), _p(v), _p(u), _p(h), theta.size, _p(off), _p(ln), _p(wd), _p(blk), ns,
                              float(lr), float(beta2), float(eps), float(lam), float(u_scale), int(t))
    return theta, v


def head_forward(H, W, b=None):
    H, W = _f64(H), _f64(W)
    b = None if b is None else _f64(b)
    N, d = H.shape
    V = W.shape[1]
    Z = np.zeros((N, V))
    _load().orc_head_forward(_p(H), N, d, _p(W), V, _p(b), _p(Z))
    return Z


def bom_step_linear_head(H, labels, theta, v, q, t, *, d, V, lr, lam, beta1, beta2, eps, segments,
                         weight_decay=0.0, ignore_index=-100):
    """One full step of Algorithm 1 for a linear softmax head whose flat parameters are
    theta = [W (d x V, row-major), b (V)]: forward, s, q / q_hat, the mixed-objective gradient
    u = [dW, db], then the second moment and the update. Returns a dict with every stage."""
    W = theta[: d * V].reshape(d, V)
    b = theta[d * V: d * V + V]
    Z = head_forward(H, W, b)
    res = residual(Z, labels, ignore_index, want_R=False)
    q_new, q_hat = ema(q, res["s"], beta1, t)
    dW = dW_cols(H, Z, labels, res["row_lse"], q_hat, res["n_valid"], lam, ignore_index=ignore_index)
    dbias = db(Z, labels, res["row_lse"], q_hat, res["n_valid"], lam, ignore_index=ignore_index)
    u = np.concatenate([dW.reshape(-1), dbias])
    theta_new, v_new = update_dense(theta, v, u, lr=lr, beta2=beta2, eps=eps, t=t, segments=segments,
                                    weight_decay=weight_decay)
    return dict(Z=Z, res=res, q=q_new, q_hat=q_hat, u=u, theta=theta_new, v=v_new)


def state_bytes(P: int, V: int, optimizer: str, bytes_per=4) -> int:
    """Parameter-shaped optimizer state in bytes: AdamW keeps m and v; BOM keeps v plus one V-vector."""
    if optimizer == "adamw":
        return 2 * P * bytes_per
    if optimizer == "bom":
        return P * bytes_per + V * bytes_per
    raise ValueError(optimizer)
