"""Thin ctypes binding of libbom.so (C-ABI in include/bom.h) with the same entry-point names.

Argument marshalling only: torch tensors supply device memory and the current HIP stream;
every step of the BOM hot path runs in the library's HIP kernels. There is no CPU or PyTorch
fallback: if libbom.so is missing or fails to load, every call raises.
"""
from __future__ import annotations

import ctypes
import os
import threading

import torch

from . import _build

BOM_OK = 0
BOM_F32, BOM_BF16 = 0, 1
BOM_FLAG_LABEL_RANGE, BOM_FLAG_EMPTY, BOM_FLAG_RESIDUAL_RECOMPUTED = 1, 2, 4
BOM_V_DENSE, BOM_V_FACTORED, BOM_V_BLOCKS = 0, 1, 2
BOM_MAX_SEGMENTS = 16

_lock = threading.Lock()
_lib = None


class BomError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"status {status}: {detail}")
        self.status = status
        self.detail = detail


class bom_segment(ctypes.Structure):
    _fields_ = [("offset", ctypes.c_int64), ("length", ctypes.c_int64), ("weight_decay", ctypes.c_float)]


class bom_update_cfg(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta2", ctypes.c_float), ("eps", ctypes.c_float), ("lambda_", ctypes.c_float),
                ("u_scale", ctypes.c_float), ("t", ctypes.c_int64), ("v_layout", ctypes.c_int32),
                ("block_rows", ctypes.c_int64), ("block_cols", ctypes.c_int64), ("clip_norm", ctypes.c_float),
                ("clip_stats", ctypes.c_void_p), ("state_dt", ctypes.c_int32),
                ("seg_blocks", ctypes.POINTER(ctypes.c_int64))]


def lib_path() -> str:
    return _build.LIB_PATH


class StaleLibraryError(RuntimeError):
    """libbom.so was built from sources other than the ones in the tree."""


def load(build_if_missing: bool = True):
    """Load libbom.so (building it in-tree only when no built library exists). A library whose build id
    (the hash of the sources it was compiled from) differs from the sources in the tree is refused: rebuild
    it with paper_2609_36738_amd._build.build() (or __graft_entry__.build())."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(_build.LIB_PATH):
            if not build_if_missing:
                raise FileNotFoundError(f"{_build.LIB_PATH} is not built")
            _build.build()
        lib = ctypes.CDLL(_build.LIB_PATH)
        lib.bom_build_id.restype = ctypes.c_char_p
        lib.bom_build_id.argtypes = []
        built, current = lib.bom_build_id().decode(), _build.source_hash()
        if built != current:
            raise StaleLibraryError(f"{_build.LIB_PATH} was built from sources {built}, the tree holds {current}: "
                                    "rebuild it")
        vp, i64, i32, f32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
        lib.bom_status_string.restype = ctypes.c_char_p
        lib.bom_status_string.argtypes = [ctypes.c_int]
        lib.bom_last_error.restype = ctypes.c_char_p
        lib.bom_last_error.argtypes = []
        lib.bom_version.restype = i32
        lib.bom_residual_workspace_bytes.restype = sz
        lib.bom_residual_workspace_bytes.argtypes = [i64, i64, ctypes.c_int]
        lib.bom_residual.restype = ctypes.c_int
        lib.bom_residual.argtypes = [vp, ctypes.c_int, i64, i64, i64, vp, i32, vp, vp, vp, vp, vp, ctypes.c_int, i64, vp,
                                     vp, vp, vp, sz, vp]
        lib.bom_residual_noalloc.restype = ctypes.c_int
        lib.bom_residual_noalloc.argtypes = [vp, ctypes.c_int, i64, i64, i64, vp, i32, vp, vp, vp, vp, vp, ctypes.c_int,
                                             i64, vp, vp, vp, vp]
        lib.bom_ema.restype = ctypes.c_int
        lib.bom_ema.argtypes = [vp, vp, i64, f32, i64, vp, vp]
        lib.bom_head_vjp_workspace_bytes.restype = sz
        lib.bom_head_vjp_workspace_bytes.argtypes = [i64, i64, i64, ctypes.c_int, ctypes.c_int]
        lib.bom_head_vjp.restype = ctypes.c_int
        lib.bom_head_vjp.argtypes = [vp, i64, vp, i64, vp, i32, i64, ctypes.c_int, i64, i64, i64, vp, i32, vp, vp, vp,
                                     vp, f32, vp, ctypes.c_int, i64, f32, vp, vp, ctypes.c_int, i64, vp, sz, vp]
        lib.bom_update_workspace_bytes.restype = sz
        lib.bom_update_workspace_bytes.argtypes = [i64, ctypes.POINTER(bom_update_cfg)]
        lib.bom_update.restype = ctypes.c_int
        lib.bom_update.argtypes = [vp, vp, vp, vp, vp, i64, ctypes.POINTER(bom_segment), i32, f32,
                                   ctypes.POINTER(bom_update_cfg), vp, sz, vp]
        lib.bom_adamw_update.restype = ctypes.c_int
        lib.bom_adamw_update.argtypes = [vp, vp, vp, vp, vp, i64, ctypes.POINTER(bom_segment), i32, f32, f32,
                                         ctypes.POINTER(bom_update_cfg), vp, sz, vp]
        lib.bom_head_telemetry_workspace_bytes.restype = sz
        lib.bom_head_telemetry_workspace_bytes.argtypes = [i64, i64, i64]
        lib.bom_head_telemetry.restype = ctypes.c_int
        lib.bom_head_telemetry.argtypes = [vp, i64, ctypes.c_int, vp, i64, ctypes.c_int, i64, i64, i64, vp, i32, vp, vp,
                                           vp, vp, i64, vp, f32, i64, vp, vp, sz, vp]
        lib.bom_head_forward_residual_workspace_bytes.restype = sz
        lib.bom_head_forward_residual_workspace_bytes.argtypes = [i64, i64, ctypes.c_int]
        lib.bom_head_forward_residual.restype = ctypes.c_int
        lib.bom_head_forward_residual.argtypes = [vp, i64, vp, i64, vp, ctypes.c_int, i64, i64, i64, vp, i64, vp, i32,
                                                  vp, vp, vp, vp, vp, i64, vp, vp, vp, vp, sz, vp]
        lib.bom_head_forward.restype = ctypes.c_int
        lib.bom_head_forward.argtypes = [vp, i64, vp, i64, vp, ctypes.c_int, i64, i64, i64, vp, i64, vp]
        _lib = lib
        return lib


def _check(st: int):
    if st != BOM_OK:
        raise BomError(st, load().bom_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return BOM_F32
    if t.dtype == torch.bfloat16:
        return BOM_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _rowmajor(t: torch.Tensor, name: str) -> int:
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError(f"{name} must be a 2-D tensor with unit column stride")
    return t.stride(0)


def _workspace(nbytes: int, device, ws):
    if nbytes == 0:
        return ws
    if ws is None or ws.numel() < nbytes:
        ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
    return ws


def bom_residual_workspace_bytes(N: int, V: int, dt: int) -> int:
    return load().bom_residual_workspace_bytes(N, V, dt)


def bom_residual(Z, labels, *, ignore_index=-100, s=None, row_lse=None, row_argmax=None, row_target=None, R=None,
                 write_R=True, loss=None, n_valid=None, flags=None, workspace=None, stream=None) -> dict:
    """Row statistics, residual rows R and the batch-mean residual s (see include/bom.h)."""
    lib = load()
    N, V = Z.shape
    dev = Z.device
    dt = _dtype_code(Z)
    ldz = _rowmajor(Z, "Z")
    if labels.dtype != torch.int32:
        raise TypeError("labels must be int32")
    s = torch.empty(V, dtype=torch.float32, device=dev) if s is None else s
    row_lse = torch.empty(N, dtype=torch.float32, device=dev) if row_lse is None else row_lse
    row_argmax = torch.empty(N, dtype=torch.int32, device=dev) if row_argmax is None else row_argmax
    row_target = torch.empty(N, dtype=torch.float32, device=dev) if row_target is None else row_target
    if R is None and write_R:
        R = torch.empty((N, V), dtype=Z.dtype, device=dev)
    ldr = _rowmajor(R, "R") if R is not None else V
    loss = torch.empty(1, dtype=torch.float32, device=dev) if loss is None else loss
    n_valid = torch.empty(1, dtype=torch.int32, device=dev) if n_valid is None else n_valid
    flags = torch.empty(1, dtype=torch.int32, device=dev) if flags is None else flags
    nb = lib.bom_residual_workspace_bytes(N, V, dt)
    workspace = _workspace(nb, dev, workspace)
    _check(lib.bom_residual(_ptr(Z), dt, N, V, ldz, _ptr(labels), ignore_index, _ptr(s), _ptr(row_lse),
                            _ptr(row_argmax), _ptr(row_target), _ptr(R), dt, ldr, _ptr(loss), _ptr(n_valid),
                            _ptr(flags), _ptr(workspace), nb if workspace is None else workspace.numel(),
                            _stream(stream)))
    return dict(s=s, row_lse=row_lse, row_argmax=row_argmax, row_target=row_target, R=R, loss=loss, n_valid=n_valid,
                flags=flags, workspace=workspace)


RESIDUAL_SCRATCH_BYTES = 64 << 20   # BOM_RESIDUAL_SCRATCH_BYTES


def bom_residual_noalloc(Z, labels, *, ignore_index=-100, s, row_lse, row_argmax=None, row_target=None, R=None,
                         loss, n_valid, flags, stream=None) -> dict:
    """bom_residual on the library's fixed scratch array (no workspace; the call allocates nothing, so every
    output tensor is passed in). Calls that overlap on one device race on the shared scratch."""
    lib = load()
    N, V = Z.shape
    dt = _dtype_code(Z)
    ldz = _rowmajor(Z, "Z")
    if labels.dtype != torch.int32:
        raise TypeError("labels must be int32")
    ldr = _rowmajor(R, "R") if R is not None else V
    _check(lib.bom_residual_noalloc(_ptr(Z), dt, N, V, ldz, _ptr(labels), ignore_index, _ptr(s), _ptr(row_lse),
                                    _ptr(row_argmax), _ptr(row_target), _ptr(R), dt, ldr, _ptr(loss), _ptr(n_valid),
                                    _ptr(flags), _stream(stream)))
    return dict(s=s, row_lse=row_lse, row_argmax=row_argmax, row_target=row_target, R=R, loss=loss, n_valid=n_valid,
                flags=flags)


def bom_ema(q, s, beta1: float, t: int, q_hat=None, stream=None):
    """q <- beta1 q + (1 - beta1) s in place; returns q_hat = q / (1 - beta1^t)."""
    lib = load()
    q_hat = torch.empty_like(q) if q_hat is None else q_hat
    _check(lib.bom_ema(_ptr(q), _ptr(s), q.numel(), float(beta1), int(t), _ptr(q_hat), _stream(stream)))
    return q_hat


def bom_head_vjp_workspace_bytes(N: int, d: int, V: int, dt: int, dw_dt: int = BOM_F32) -> int:
    return load().bom_head_vjp_workspace_bytes(N, d, V, dt, dw_dt)


def bom_head_vjp(H, W, R, labels, q_hat, n_valid, *, s=None, lam=0.5, ignore_index=-100, dW=None, dW_beta=0.0,
                 want_db=False, db=None, want_dH=True, dH=None, dh_dtype=None, workspace=None, stream=None,
                 row_lse=None) -> dict:
    """dW = H^T G, db = (1 - lambda) s + lambda q_hat, dH = G W^T with G folded from R and q_hat.
    With row_lse given, the third argument is the logits Z (is_residual = 0) and the kernels form R
    from Z and row_lse themselves."""
    lib = load()
    N, d = H.shape
    V = W.shape[1]
    dev = H.device
    dt = _dtype_code(H)
    if _dtype_code(W) != dt or _dtype_code(R) != dt:
        raise TypeError("H, W and R (or Z) must share a dtype")
    if row_lse is not None and (row_lse.dtype != torch.float32 or row_lse.numel() != N or not row_lse.is_contiguous()):
        raise ValueError("row_lse must be a contiguous float32 tensor of N elements")
    ldh, ldw, ldr = _rowmajor(H, "H"), _rowmajor(W, "W"), _rowmajor(R, "R")
    dW = torch.empty((d, V), dtype=torch.float32, device=dev) if dW is None else dW
    lddw = _rowmajor(dW, "dW")
    dw_dt = _dtype_code(dW)
    if want_db and db is None:
        db = torch.empty(V, dtype=dW.dtype, device=dev)
    if db is not None and db.dtype != dW.dtype:
        raise TypeError("db must have dW's dtype")
    if want_dH and dH is None:
        dH = torch.empty((N, d), dtype=dh_dtype or H.dtype, device=dev)
    dh_dt = _dtype_code(dH) if dH is not None else BOM_F32
    lddh = _rowmajor(dH, "dH") if dH is not None else d
    nb = lib.bom_head_vjp_workspace_bytes(N, d, V, dt, dw_dt)
    workspace = _workspace(nb, dev, workspace)
    _check(lib.bom_head_vjp(_ptr(H), ldh, _ptr(W), ldw, _ptr(R), 0 if row_lse is not None else 1, ldr, dt, N, d, V,
                            _ptr(labels), ignore_index, _ptr(row_lse),
                            _ptr(q_hat), _ptr(s), _ptr(n_valid), float(lam), _ptr(dW), dw_dt, lddw, float(dW_beta),
                            _ptr(db),
                            _ptr(dH), dh_dt, lddh, _ptr(workspace), 0 if workspace is None else workspace.numel(),
                            _stream(stream)))
    return dict(dW=dW, db=db, dH=dH, workspace=workspace)


def make_update_cfg(*, lr, beta2, eps, t, lam=0.5, u_scale=1.0, factored=False, block_rows=4096, block_cols=4096,
                    clip_norm=0.0, clip_stats=None, state_dtype=torch.float32, blocks=None):
    """clip_norm > 0 turns on global-norm clipping; clip_stats (a device fp32 tensor of 2) receives the
    numerator's norm before clipping and the factor. state_dtype torch.bfloat16 selects bf16 storage
    of theta, v, u and h (dense layout). blocks (one block length per segment) selects the block-shared
    second moment; the segments passed to bom_update must then tile the buffer in order."""
    if factored and blocks is not None:
        raise ValueError("choose the factored or the block layout, not both")
    if state_dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("state_dtype must be torch.float32 or torch.bfloat16")
    if clip_stats is not None and (clip_stats.dtype != torch.float32 or not clip_stats.is_cuda or
                                   clip_stats.numel() < 2 or not clip_stats.is_contiguous()):
        raise ValueError("clip_stats must be a contiguous device float32 tensor of at least 2 elements")
    layout = BOM_V_FACTORED if factored else (BOM_V_BLOCKS if blocks is not None else BOM_V_DENSE)
    cfg = bom_update_cfg(lr, beta2, eps, lam, u_scale, int(t), layout, block_rows, block_cols, float(clip_norm),
                         None if clip_stats is None else clip_stats.data_ptr(),
                         BOM_BF16 if state_dtype == torch.bfloat16 else BOM_F32)
    if blocks is not None:
        arr = (ctypes.c_int64 * max(1, len(blocks)))(*[int(b) for b in blocks])
        cfg.seg_blocks = ctypes.cast(arr, ctypes.POINTER(ctypes.c_int64))
        cfg._blocks = arr   # keeps the host array alive with the struct
        cfg._nblocks = len(blocks)
    return cfg


def blocks_count(segments, blocks) -> int:
    """Entries of the block-shared second moment for these segments and block lengths."""
    return int(sum(-(-int(s[1]) // int(b)) for s, b in zip(segments, blocks)))


def bom_update_workspace_bytes(P: int, cfg: bom_update_cfg) -> int:
    return load().bom_update_workspace_bytes(P, ctypes.byref(cfg))


def bom_update(theta, v, u, cfg: bom_update_cfg, *, v_col=None, h=None, segments=(), weight_decay=0.0,
               workspace=None, stream=None):
    """theta and v (or the factored Rr = v, Cc = v_col) updated in place; see include/bom.h."""
    lib = load()
    P = theta.numel()
    want = torch.bfloat16 if cfg.state_dt == BOM_BF16 else torch.float32
    blocks = cfg.v_layout == BOM_V_BLOCKS
    for name, x in (("theta", theta), ("u", u), ("h", h)) + ((("v", v),) if v_col is None and not blocks else ()):
        if x is not None and (x.dtype != want or not x.is_contiguous() or x.numel() != P):
            raise ValueError(f"{name} must be a contiguous {want} tensor of {P} elements")
    if blocks:
        if getattr(cfg, "_nblocks", -1) != len(segments):
            raise ValueError("the block layout needs one block length per segment")
        nv = blocks_count(segments, list(cfg._blocks)[:len(segments)])
        if v.dtype != torch.float32 or not v.is_contiguous() or v.numel() != nv:
            raise ValueError(f"v must be a contiguous float32 tensor of {nv} block entries")
    segs = (bom_segment * max(1, len(segments)))(*[bom_segment(int(o), int(n), float(w)) for o, n, w in segments])
    nb = lib.bom_update_workspace_bytes(P, ctypes.byref(cfg))
    workspace = _workspace(nb, theta.device, workspace)
    _check(lib.bom_update(_ptr(theta), _ptr(v), _ptr(v_col), _ptr(u), _ptr(h), P, segs, len(segments),
                          float(weight_decay), ctypes.byref(cfg), _ptr(workspace),
                          0 if workspace is None else workspace.numel(), _stream(stream)))
    return workspace


def bom_adamw_update(theta, m, v, g, cfg: bom_update_cfg, *, beta1=0.9, v_col=None, segments=(), weight_decay=0.0,
                     workspace=None, stream=None):
    """AdamW (the comparison optimizer) in place: theta, m and v (or the factored Rr = v, Cc = v_col)."""
    lib = load()
    P = theta.numel()
    for name, x in (("theta", theta), ("m", m), ("g", g)) + ((("v", v),) if v_col is None else ()):
        if x.dtype != torch.float32 or not x.is_contiguous() or x.numel() != P:
            raise ValueError(f"{name} must be a contiguous float32 tensor of {P} elements")
    segs = (bom_segment * max(1, len(segments)))(*[bom_segment(int(o), int(n), float(w)) for o, n, w in segments])
    nb = lib.bom_update_workspace_bytes(P, ctypes.byref(cfg))
    workspace = _workspace(nb, theta.device, workspace)
    _check(lib.bom_adamw_update(_ptr(theta), _ptr(m), _ptr(v), _ptr(v_col), _ptr(g), P, segs, len(segments),
                                float(weight_decay), float(beta1), ctypes.byref(cfg), _ptr(workspace),
                                0 if workspace is None else workspace.numel(), _stream(stream)))
    return workspace


TELEMETRY_FIELDS = ("cos", "drift", "cancellation", "m_norm", "h_norm")


def bom_head_telemetry(H, R, labels, s, q_hat, n_valid, M_W, *, beta1, t, M_b=None, out=None, ignore_index=-100,
                       workspace=None, stream=None) -> dict:
    """Drift telemetry of the linear head (M_W, M_b updated in place); out (device fp32 [5]) holds
    TELEMETRY_FIELDS. Returns dict(out=..., workspace=...)."""
    lib = load()
    N, d = H.shape
    V = R.shape[1]
    if M_W.dtype != torch.float32 or tuple(M_W.shape) != (d, V) or (M_b is not None and M_b.dtype != torch.float32):
        raise ValueError("M_W must be fp32 [d, V] and M_b fp32 [V]")
    out = torch.zeros(5, dtype=torch.float32, device=H.device) if out is None else out
    nb = lib.bom_head_telemetry_workspace_bytes(N, d, V)
    workspace = _workspace(nb, H.device, workspace)
    _check(lib.bom_head_telemetry(_ptr(H), _rowmajor(H, "H"), _dtype_code(H), _ptr(R), _rowmajor(R, "R"), _dtype_code(R),
                                  N, d, V, _ptr(labels), ignore_index, _ptr(s), _ptr(q_hat), _ptr(n_valid), _ptr(M_W),
                                  _rowmajor(M_W, "M_W"), _ptr(M_b), float(beta1), int(t), _ptr(out), _ptr(workspace),
                                  0 if workspace is None else workspace.numel(), _stream(stream)))
    return dict(out=out, workspace=workspace)


def bom_head_forward(H, W, b=None, Z=None, stream=None):
    """Support call: Z = H W (+ b), fp32."""
    lib = load()
    N, d = H.shape
    V = W.shape[1]
    Z = torch.empty((N, V), dtype=H.dtype, device=H.device) if Z is None else Z
    _check(lib.bom_head_forward(_ptr(H), _rowmajor(H, "H"), _ptr(W), _rowmajor(W, "W"), _ptr(b), _dtype_code(H), N, d,
                                V, _ptr(Z), _rowmajor(Z, "Z"), _stream(stream)))
    return Z


def bom_head_forward_residual(H, W, labels, *, b=None, Z=None, ignore_index=-100, R=None, write_R=True, out=None,
                              workspace=None, stream=None) -> dict:
    """Z = H W (+ b) and the residual outputs of bom_residual on it, in one call (the forward's epilogue
    reduces each row's tiles on the matrix-core path). out: a dict of preallocated outputs to reuse."""
    lib = load()
    N, d = H.shape
    V = W.shape[1]
    dev = H.device
    dt = _dtype_code(H)
    o = dict(out or {})
    Z = Z if Z is not None else o.get("Z", torch.empty((N, V), dtype=H.dtype, device=dev))
    if R is None and write_R:
        R = o.get("R", torch.empty((N, V), dtype=H.dtype, device=dev))
    res = dict(Z=Z, R=R)
    for k, shape, dtype in (("s", (V,), torch.float32), ("row_lse", (N,), torch.float32),
                            ("row_argmax", (N,), torch.int32), ("row_target", (N,), torch.float32),
                            ("loss", (1,), torch.float32), ("n_valid", (1,), torch.int32), ("flags", (1,), torch.int32)):
        res[k] = o.get(k, torch.empty(shape, dtype=dtype, device=dev))
    nb = lib.bom_head_forward_residual_workspace_bytes(N, V, dt)
    workspace = _workspace(nb, dev, workspace)
    _check(lib.bom_head_forward_residual(_ptr(H), _rowmajor(H, "H"), _ptr(W), _rowmajor(W, "W"), _ptr(b), dt, N, d, V,
                                         _ptr(Z), _rowmajor(Z, "Z"), _ptr(labels), ignore_index, _ptr(res["s"]),
                                         _ptr(res["row_lse"]), _ptr(res["row_argmax"]), _ptr(res["row_target"]), _ptr(R),
                                         _rowmajor(R, "R") if R is not None else V, _ptr(res["loss"]),
                                         _ptr(res["n_valid"]), _ptr(res["flags"]), _ptr(workspace),
                                         0 if workspace is None else workspace.numel(), _stream(stream)))
    res["workspace"] = workspace
    return res
