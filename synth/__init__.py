"""Seeded synthetic inputs for the BOM hot path (shared by tests, bench and smoke).

This module holds no arithmetic of the method. It wraps ``synth.c`` (Philox4x32-10
counter-based generator, Box-Muller normals, uniform and truncated-Zipf labels) and
the workload table in :mod:`synth.workloads`. Every tensor is addressed by
(seed, stream id, element index), so any slice can be regenerated on its own.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.c")
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lock = threading.Lock()
_lib = None

BASE_SEED = 1234
# Stream ids (one per tensor kind); per-step tensors add the step index.
STREAM_H = 1
STREAM_W = 2
STREAM_LABELS = 3
STREAM_THETA = 4
STREAM_V0 = 5
STREAM_IGNORE = 6
STREAM_U = 16      # + step
STREAM_Z = 64      # + step
STREAM_SPLIT_H = 112  # + step: the history half in split-numerator mode


def build() -> str:
    """Compile libsynth.so with gcc (OpenMP); returns its path."""
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
        i64, u64, u32, f64, vp = ctypes.c_int64, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_double, ctypes.c_void_p
        lib.synth_philox.argtypes = [u32, u32, u32, u32, u32, u32, vp]
        lib.synth_normal_f32.argtypes = [vp, i64, i64, u64, u32, f64]
        lib.synth_normal_bf16.argtypes = [vp, i64, i64, u64, u32, f64]
        lib.synth_labels_uniform.argtypes = [vp, i64, i64, u64, u32, i64]
        lib.synth_labels_zipf.argtypes = [vp, i64, i64, u64, u32, i64, f64]
        lib.synth_labels_zipf.restype = ctypes.c_int
        lib.synth_uniform_f64.argtypes = [vp, i64, i64, u64, u32]
        lib.synth_bf16_to_f32.argtypes = [vp, vp, i64]
        _lib = lib
        return lib


def _ptr(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


def philox(counter, key) -> tuple:
    """Raw Philox4x32-10 block for a 4-word counter and 2-word key."""
    out = np.zeros(4, np.uint32)
    _load().synth_philox(*[int(c) for c in counter], *[int(k) for k in key], _ptr(out))
    return tuple(int(x) for x in out)


def normal_f32(n: int, stream: int, std: float, start: int = 0, seed: int = BASE_SEED, out=None) -> np.ndarray:
    out = np.empty(n, np.float32) if out is None else out
    _load().synth_normal_f32(_ptr(out), n, start, seed, stream, float(std))
    return out


def normal_bf16(n: int, stream: int, std: float, start: int = 0, seed: int = BASE_SEED, out=None) -> np.ndarray:
    """bf16 normals as raw uint16 bit patterns."""
    out = np.empty(n, np.uint16) if out is None else out
    _load().synth_normal_bf16(_ptr(out), n, start, seed, stream, float(std))
    return out


def labels_uniform(n: int, C: int, stream: int = STREAM_LABELS, start: int = 0, seed: int = BASE_SEED) -> np.ndarray:
    out = np.empty(n, np.int32)
    _load().synth_labels_uniform(_ptr(out), n, start, seed, stream, C)
    return out


def labels_zipf(n: int, V: int, a: float = 1.1, stream: int = STREAM_LABELS, start: int = 0,
                seed: int = BASE_SEED) -> np.ndarray:
    out = np.empty(n, np.int32)
    rc = _load().synth_labels_zipf(_ptr(out), n, start, seed, stream, V, float(a))
    if rc != 0:
        raise MemoryError("synth_labels_zipf: allocation failed")
    return out


def uniform_f64(n: int, stream: int, start: int = 0, seed: int = BASE_SEED) -> np.ndarray:
    out = np.empty(n, np.float64)
    _load().synth_uniform_f64(_ptr(out), n, start, seed, stream)
    return out


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    out = np.empty(bits.shape, np.float32)
    _load().synth_bf16_to_f32(_ptr(bits), _ptr(out), bits.size)
    return out


def with_ignored(labels: np.ndarray, frac: float, ignore_index: int = -100, stream: int = STREAM_IGNORE,
                 seed: int = BASE_SEED) -> np.ndarray:
    """Copy of ``labels`` with a seeded fraction set to ``ignore_index``."""
    u = uniform_f64(labels.size, stream, seed=seed)
    out = labels.copy()
    out[u <= frac] = ignore_index
    return out
