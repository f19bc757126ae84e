"""Helpers for the GPU parity tests: seeded inputs (from synth) on host and device, oracle calls on
the same inputs, and the comparison bars (bit-exact for integers, relative bounds for floats)."""
import os
import sys

import numpy as np
import pytest
import torch

import synth

ON_GPU = torch.cuda.is_available()
needs_gpu = pytest.mark.skipif(not ON_GPU, reason="needs an MI355X")


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def dev():
    return torch.device("cuda:0")


def bf16_tensor(bits: np.ndarray, shape) -> torch.Tensor:
    """uint16 bf16 patterns -> device bfloat16 tensor (exact)."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).reshape(shape)
    return t.to(dev())


def to_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def gen_matrix(n_rows, n_cols, stream, std, dtype, start=0):
    """(host fp32 exact image, device tensor) of a seeded N(0, std) matrix."""
    n = n_rows * n_cols
    if dtype == "bf16":
        bits = synth.normal_bf16(n, stream, std, start=start)
        host = synth.bf16_to_f32(bits).reshape(n_rows, n_cols)
        return host, bf16_tensor(bits, (n_rows, n_cols))
    host = synth.normal_f32(n, stream, std, start=start).reshape(n_rows, n_cols)
    return host, torch.from_numpy(host).to(dev())


def gen_labels(N, V, kind, ignore_frac=0.0, n_out_of_range=0):
    y = synth.labels_uniform(N, V) if kind == "uniform" else synth.labels_zipf(N, V)
    if ignore_frac > 0:
        y = synth.with_ignored(y, ignore_frac)
    if n_out_of_range:
        idx = np.linspace(1, N - 2, n_out_of_range).astype(int)
        y[idx[::2]] = V
        y[idx[1::2]] = -7
    return y


def rel_fro(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


def check_s(s_gpu, orc, R_oracle_pmean=None, tol=1e-5):
    """Norm-wise and condition-aware per-element bound on s:
    |ds_j| <= tol * (mean_i p_ij + count_j / N_t) + tiny."""
    s_o = orc["s"]
    assert rel_fro(s_gpu, s_o) <= tol, rel_fro(s_gpu, s_o)
    if R_oracle_pmean is not None:
        bound = tol * R_oracle_pmean + 1e-12
        assert (np.abs(s_gpu - s_o) <= bound).all(), np.max(np.abs(s_gpu - s_o) / bound)
