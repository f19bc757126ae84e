"""Pins of the fp64 oracle against what the paper and the mathematics fix (CPU only).

Each test checks the oracle against something other than itself: library routines
(scipy's softmax / logsumexp), brute-force per-example Jacobians, finite differences,
closed forms, explicit EMA sums, Lemma 2, numbers the paper prints (tests/golden), and
the linear-model equivalence of BOM and the own-step control.
"""
import math

import numpy as np
import pytest
from scipy.special import log_softmax, logsumexp, softmax

import oracle
from conftest import read_golden

LAM, B1, B2, EPS = 0.5, 0.9, 0.999, 1e-8


def _rng(seed=0):
    return np.random.default_rng(seed)


def _head_problem(N=4, d=3, V=5, seed=0, scale=1.0):
    r = _rng(seed)
    H = r.standard_normal((N, d))
    W = r.standard_normal((d, V)) * 0.5 * scale
    b = r.standard_normal(V) * 0.1
    y = r.integers(0, V, N).astype(np.int32)
    return H, W, b, y


# ----------------------------------------------------------------------------- residual

def test_residual_matches_library_softmax():
    r = _rng(1)
    Z = r.standard_normal((37, 23)) * 3
    y = r.integers(0, 23, 37).astype(np.int32)
    out = oracle.residual(Z, y)
    P = softmax(Z, axis=1)
    Y = np.eye(23)[y]
    np.testing.assert_allclose(out["row_lse"], logsumexp(Z, axis=1), rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(out["R"], P - Y, atol=1e-14)
    np.testing.assert_allclose(out["s"], (P - Y).mean(0), atol=1e-15)
    np.testing.assert_allclose(out["loss"], -log_softmax(Z, axis=1)[np.arange(37), y].mean(), rtol=1e-14)
    assert (out["row_argmax"] == Z.argmax(1)).all()
    assert (out["row_target"] == Z[np.arange(37), y]).all()
    assert out["n_valid"] == 37 and out["flags"] == 0


def test_residual_rows_and_s_sum_to_zero():
    # Sec. 3.1: every softmax residual has zero coordinate sum, hence so do s and q.
    r = _rng(2)
    Z = r.standard_normal((50, 31)) * 5
    y = r.integers(0, 31, 50).astype(np.int32)
    out = oracle.residual(Z, y)
    assert np.abs(out["R"].sum(1)).max() < 1e-14
    assert abs(out["s"].sum()) < 1e-15
    q = np.zeros(31)
    for t in range(1, 6):
        q, qh = oracle.ema(q, out["s"] * t, B1, t)
        assert abs(q.sum()) < 1e-14 and abs(qh.sum()) < 1e-14


def test_uniform_logits_closed_form():
    # z_ij = c: p = 1/V, CE = ln V, lse = c + ln V, s_j = 1/V - count_j / N_t, argmax = 0.
    N, V, c = 40, 7, 0.375
    y = _rng(3).integers(0, V, N).astype(np.int32)
    out = oracle.residual(np.full((N, V), c), y)
    cnt = np.bincount(y, minlength=V)
    np.testing.assert_allclose(out["s"], 1.0 / V - cnt / N, atol=1e-15)
    assert abs(out["loss"] - math.log(V)) < 1e-14
    np.testing.assert_allclose(out["row_lse"], c + math.log(V), rtol=1e-15)
    assert (out["row_argmax"] == 0).all()


def test_residual_is_gradient_of_mean_ce():
    # Finite differences: d(mean CE)/dz_ij = r_ij / N_t (central differences, fp64).
    r = _rng(4)
    N, V = 6, 9
    Z = r.standard_normal((N, V)) * 2
    y = r.integers(0, V, N).astype(np.int32)
    y[2] = -100
    out = oracle.residual(Z, y)
    h = 1e-6
    for i in range(N):
        for j in range(V):
            Zp, Zm = Z.copy(), Z.copy()
            Zp[i, j] += h
            Zm[i, j] -= h
            fd = (oracle.residual(Zp, y, want_R=False)["loss"] - oracle.residual(Zm, y, want_R=False)["loss"]) / (2 * h)
            assert abs(fd - out["R"][i, j] / out["n_valid"]) < 1e-8


def test_argmax_ties_take_lowest_index():
    Z = np.array([[1.0, 3.0, 3.0, 0.0], [2.0, 2.0, 2.0, 2.0], [-1.0, -5.0, -1.0, -1.0]])
    out = oracle.residual(Z, np.array([0, 1, 2], np.int32))
    assert list(out["row_argmax"]) == [1, 0, 0]


def test_ignored_and_out_of_range_labels():
    r = _rng(5)
    N, V = 20, 6
    Z = r.standard_normal((N, V))
    y = r.integers(0, V, N).astype(np.int32)
    y[[1, 7]] = -100
    y[4] = V          # out of range
    y[9] = -3         # out of range
    out = oracle.residual(Z, y)
    keep = np.array([i not in (1, 7, 4, 9) for i in range(N)])
    P = softmax(Z[keep], axis=1)
    Y = np.eye(V)[y[keep]]
    np.testing.assert_allclose(out["s"], (P - Y).mean(0), atol=1e-15)
    assert out["n_valid"] == keep.sum()
    assert out["flags"] == oracle.FLAG_LABEL_RANGE
    assert (out["R"][~keep] == 0).all() and (out["row_target"][~keep] == 0).all()
    np.testing.assert_allclose(out["row_lse"], logsumexp(Z, axis=1), rtol=1e-14)


def test_all_rows_ignored_is_empty():
    Z = _rng(6).standard_normal((5, 4))
    y = np.full(5, -100, np.int32)
    out = oracle.residual(Z, y)
    assert out["flags"] == oracle.FLAG_EMPTY and out["n_valid"] == 0
    assert (out["s"] == 0).all() and out["loss"] == 0
    H = _rng(7).standard_normal((5, 3))
    qh = _rng(8).standard_normal(4)
    assert (oracle.dW_cols(H, Z, y, out["row_lse"], qh, 0, LAM) == 0).all()
    assert (oracle.db(Z, y, out["row_lse"], qh, 0, LAM) == 0).all()
    assert (oracle.dH_rows(_rng(9).standard_normal((3, 4)), Z, y, out["row_lse"], qh, 0, LAM) == 0).all()


# ----------------------------------------------------------------------------- EMA

def test_ema_explicit_sum_and_lemma2():
    # q_t = sum_tau w_{t,tau} s_tau with w = (1-b1) b1^(t-tau) (Sec. 3 notation); Lemma 2:
    # normalised weights sum to 1 and ||q_hat_t - s_t|| <= sum alpha_{t,tau} ||s_tau - s_t||.
    r = _rng(10)
    V, T = 11, 25
    S = r.standard_normal((T, V))
    q = np.zeros(V)
    for t in range(1, T + 1):
        q, qh = oracle.ema(q, S[t - 1], B1, t)
        w = np.array([(1 - B1) * B1 ** (t - tau) for tau in range(1, t + 1)])
        np.testing.assert_allclose(q, w @ S[:t], atol=1e-14)
        alpha = w / (1 - B1 ** t)
        assert abs(alpha.sum() - 1) < 1e-14
        np.testing.assert_allclose(qh, alpha @ S[:t], atol=1e-14)
        bound = sum(alpha[k] * np.linalg.norm(S[k] - S[t - 1]) for k in range(t))
        assert np.linalg.norm(qh - S[t - 1]) <= bound + 1e-12


def test_ema_constant_signal_and_beta_zero():
    s = _rng(11).standard_normal(8)
    q = np.zeros(8)
    for t in range(1, 12):
        q, qh = oracle.ema(q, s, B1, t)
        np.testing.assert_allclose(qh, s, rtol=1e-13)
    q = _rng(12).standard_normal(8)
    _, qh = oracle.ema(q, s, 0.0, 5)
    assert (qh == s).all()


def test_binary_history_is_one_scalar():
    # Sec. 3.1: V = 2 gives q_t = (a_t, -a_t).
    r = _rng(13)
    q = np.zeros(2)
    for t in range(1, 8):
        Z = r.standard_normal((16, 2)) * 2
        y = r.integers(0, 2, 16).astype(np.int32)
        s = oracle.residual(Z, y)["s"]
        q, qh = oracle.ema(q, s, B1, t)
        assert abs(q[0] + q[1]) < 1e-16 and abs(qh[0] + qh[1]) < 1e-15


# ----------------------------------------------------------------------------- head VJP

def _jacobians(H, W, b):
    """Brute-force per-example Jacobians of z_i = W^T h_i + b with respect to theta = (W, b, H),
    by central differences of numpy's forward map (exact for a linear map up to rounding)."""
    N, d = H.shape
    V = W.shape[1]
    theta = np.concatenate([W.ravel(), b, H.ravel()])

    def fwd(th):
        Wt = th[: d * V].reshape(d, V)
        bt = th[d * V: d * V + V]
        Ht = th[d * V + V:].reshape(N, d)
        return Ht @ Wt + bt

    J = np.zeros((N, V, theta.size))
    h = 1e-3
    for p in range(theta.size):
        tp, tm = theta.copy(), theta.copy()
        tp[p] += h
        tm[p] -= h
        J[:, :, p] = (fwd(tp) - fwd(tm)) / (2 * h)
    return J


def _oracle_u(H, W, b, y, q_hat, lam):
    Z = H @ W + b
    res = oracle.residual(Z, y)
    nv = res["n_valid"]
    dW = oracle.dW_cols(H, Z, y, res["row_lse"], q_hat, nv, lam)
    dbias = oracle.db(Z, y, res["row_lse"], q_hat, nv, lam)
    dH = oracle.dH_rows(W, Z, y, res["row_lse"], q_hat, nv, lam)
    return np.concatenate([dW.ravel(), dbias, dH.ravel()]), res


def test_batch_decomposition_brute_force():
    # Eq. (1): g = Jbar^T s + c with c = mean (J_i - Jbar)^T (r_i - s); and Eq. (4):
    # u = (1 - lam) g + lam Jbar^T q_hat, from per-example Jacobians built by brute force.
    H, W, b, y = _head_problem(N=4, d=3, V=5, seed=14)
    J = _jacobians(H, W, b)
    q_hat = _rng(15).standard_normal(5) * 0.1
    q_hat -= q_hat.mean()
    g, res = _oracle_u(H, W, b, y, q_hat, 0.0)
    Rm = res["R"]
    s = res["s"]
    Jbar = J.mean(0)
    c = np.mean([(J[i] - Jbar).T @ (Rm[i] - s) for i in range(4)], axis=0)
    g_bf = np.mean([J[i].T @ Rm[i] for i in range(4)], axis=0)
    np.testing.assert_allclose(g, g_bf, atol=1e-9)
    np.testing.assert_allclose(g, Jbar.T @ s + c, atol=1e-9)
    u, _ = _oracle_u(H, W, b, y, q_hat, LAM)
    np.testing.assert_allclose(u, (1 - LAM) * g + LAM * Jbar.T @ q_hat, atol=1e-9)


def test_beta_zero_history_is_current_projection():
    # beta1 = 0 gives q_hat = s, so the history term is h = Jbar^T s.
    H, W, b, y = _head_problem(N=4, d=3, V=5, seed=16)
    J = _jacobians(H, W, b)
    res = oracle.residual(H @ W + b, y)
    _, qh = oracle.ema(_rng(17).standard_normal(5), res["s"], 0.0, 3)
    u1, _ = _oracle_u(H, W, b, y, qh, 1.0)
    np.testing.assert_allclose(u1, J.mean(0).T @ res["s"], atol=1e-9)


def test_head_vjp_finite_differences_of_mixed_objective():
    # Eq. (3) with q_hat detached: L_mix = (1-lam) mean CE + (lam/N) sum <z_i, q_hat>.
    H, W, b, y = _head_problem(N=6, d=4, V=7, seed=18)
    y[3] = -100
    q_hat = _rng(19).standard_normal(7) * 0.2
    valid = y != -100

    def lmix(Wt, bt, Ht):
        Z = Ht @ Wt + bt
        ls = log_softmax(Z[valid], axis=1)
        ce = -ls[np.arange(valid.sum()), y[valid]].mean()
        return (1 - LAM) * ce + LAM * (Z[valid] @ q_hat).mean()

    u, _ = _oracle_u(H, W, b, y, q_hat, LAM)
    fd = []
    h = 1e-6
    for arr_idx, shape in ((0, W.shape), (1, b.shape), (2, H.shape)):
        for k in range(int(np.prod(shape))):
            args_p = [W.copy(), b.copy(), H.copy()]
            args_m = [W.copy(), b.copy(), H.copy()]
            args_p[arr_idx].reshape(-1)[k] += h
            args_m[arr_idx].reshape(-1)[k] -= h
            fd.append((lmix(*args_p) - lmix(*args_m)) / (2 * h))
    np.testing.assert_allclose(u, np.array(fd), atol=2e-8)


def test_lambda_zero_is_textbook_softmax_ce_backward():
    H, W, b, y = _head_problem(N=9, d=5, V=6, seed=20)
    Z = H @ W + b
    res = oracle.residual(Z, y)
    qh = _rng(21).standard_normal(6)
    dW = oracle.dW_cols(H, Z, y, res["row_lse"], qh, res["n_valid"], 0.0)
    dH = oracle.dH_rows(W, Z, y, res["row_lse"], qh, res["n_valid"], 0.0)
    G = (softmax(Z, axis=1) - np.eye(6)[y]) / 9
    np.testing.assert_allclose(dW, H.T @ G, atol=1e-15)
    np.testing.assert_allclose(dH, G @ W.T, atol=1e-15)


def test_head_vjp_invariants_and_bias_identity():
    # Bias Jacobian is the identity: db = (1 - lam) s + lam q_hat exactly; zero-sum residuals and a
    # zero-sum q_hat make every dW row sum vanish and 1^T db = 0.
    H, W, b, y = _head_problem(N=30, d=8, V=12, seed=22)
    Z = H @ W + b
    res = oracle.residual(Z, y)
    q = np.zeros(12)
    for t in range(1, 4):
        q, qh = oracle.ema(q, res["s"] * (1 + 0.1 * t), B1, t)
    dW = oracle.dW_cols(H, Z, y, res["row_lse"], qh, res["n_valid"], LAM)
    dbias = oracle.db(Z, y, res["row_lse"], qh, res["n_valid"], LAM)
    np.testing.assert_allclose(dbias, (1 - LAM) * res["s"] + LAM * qh, atol=1e-16)
    assert np.abs(dW.sum(1)).max() < 1e-15
    assert abs(dbias.sum()) < 1e-16
    # linear-head closed form of the history term: Jbar^T q_hat = hbar q_hat^T for W
    dW0 = oracle.dW_cols(H, Z, y, res["row_lse"], qh, res["n_valid"], 0.0)
    np.testing.assert_allclose(dW - (1 - LAM) * dW0, LAM * np.outer(H.mean(0), qh), atol=1e-15)


def test_binary_history_direction_is_mean_margin_gradient():
    # Sec. 3.1: for V = 2, Jbar^T q_hat = a (grad of the batch-mean margin z_1 - z_2).
    H, W, b, y = _head_problem(N=10, d=4, V=2, seed=23)
    Z = H @ W + b
    res = oracle.residual(Z, y)
    _, qh = oracle.ema(np.zeros(2), res["s"], B1, 1)
    dW1 = oracle.dW_cols(H, Z, y, res["row_lse"], qh, res["n_valid"], 1.0)
    margin_grad_W = np.stack([H.mean(0), -H.mean(0)], axis=1)
    np.testing.assert_allclose(dW1, qh[0] * margin_grad_W, atol=1e-15)


def test_u_decomposition_bias_corrected_exact():
    # Classifier-history appendix with Gamma = I: u = (1-lam) g + lam (1-b1)/(1-b1^t) Jbar^T s_t
    #   + lam b1/(1-b1^t) Jbar^T q_{t-1}; and the printed 0.55 / 0.45 / 0.5 weights of Eq. (5).
    gold = read_golden("temporal_kernel.txt")
    lam, b1 = gold["lambda"], gold["beta1"]
    H, W, b, y = _head_problem(N=5, d=3, V=4, seed=24)
    J = _jacobians(H, W, b)
    Jbar = J.mean(0)
    q_prev = _rng(25).standard_normal(4) * 0.1
    q_prev -= q_prev.mean()
    for t in (2, 3, 7, 400):
        g, res = _oracle_u(H, W, b, y, np.zeros(4), 0.0)
        s = res["s"]
        _, qh = oracle.ema(q_prev, s, b1, t)
        u, _ = _oracle_u(H, W, b, y, qh, lam)
        bc = 1 - b1 ** t
        np.testing.assert_allclose(u, (1 - lam) * g + lam * (1 - b1) / bc * Jbar.T @ s
                                   + lam * b1 / bc * Jbar.T @ q_prev, atol=1e-9)
        if t == 400:  # bias correction negligible: Eq. (5) weights
            Rm = res["R"]
            c = np.mean([(J[i] - Jbar).T @ (Rm[i] - s) for i in range(5)], axis=0)
            np.testing.assert_allclose(u, gold["current_weight"] * Jbar.T @ s + gold["covariance_weight"] * c
                                       + gold["history_weight"] * Jbar.T @ q_prev, atol=1e-9)


def test_temporal_kernel_matches_printed_coefficients():
    # Full-kernel appendix: with the batch-mean signal of a fixed linear model, the coefficient of
    # Jbar^T s_t is 0.5 + 0.05/(1 - 0.9^t) and of lag k is 0.05 0.9^k / (1 - 0.9^t).
    gold = read_golden("temporal_kernel.txt")
    r = _rng(26)
    V, T = 6, 9
    S = r.standard_normal((T, V))
    q = np.zeros(V)
    for t in range(1, T + 1):
        q, qh = oracle.ema(q, S[t - 1], gold["beta1"], t)
    lam = gold["lambda"]
    bc = 1 - gold["kernel_decay"] ** T
    coef_now = gold["kernel_current_base"] + gold["kernel_scale"] / bc
    mix = (1 - lam) * S[T - 1] + lam * qh   # batch-mean part of u, in task space
    expect = coef_now * S[T - 1] + sum(gold["kernel_scale"] * gold["kernel_decay"] ** k / bc * S[T - 1 - k]
                                       for k in range(1, T))
    np.testing.assert_allclose(mix, expect, atol=1e-14)


# ----------------------------------------------------------------------------- update

def test_dense_update_first_step_closed_form():
    # t = 1: v_hat = u^2, so theta_1 = (1 - lr wd) theta - lr u / (|u| + eps).
    r = _rng(27)
    P = 1000
    th, u = r.standard_normal(P), r.standard_normal(P) * 1e-3
    u[:5] = 0.0
    segs = [(0, 600, 0.01), (600, 100, 0.0)]
    t1, v1 = oracle.update_dense(th, np.zeros(P), u, lr=1e-2, beta2=B2, eps=EPS, t=1, segments=segs,
                                 weight_decay=0.1)
    wd = np.r_[np.full(600, 0.01), np.zeros(100), np.full(300, 0.1)]
    np.testing.assert_allclose(t1, (1 - 1e-2 * wd) * th - 1e-2 * u / (np.abs(u) + EPS), rtol=1e-13, atol=1e-16)
    np.testing.assert_allclose(v1, (1 - B2) * u * u, rtol=1e-15)


def test_dense_update_second_moment_explicit_sum():
    r = _rng(28)
    P, T = 64, 6
    U = r.standard_normal((T, P))
    th = r.standard_normal(P)
    v = np.zeros(P)
    for t in range(1, T + 1):
        th_prev = th
        th, v = oracle.update_dense(th, v, U[t - 1], lr=1e-3, beta2=B2, eps=EPS, t=t)
        expect_v = sum((1 - B2) * B2 ** (t - tau) * U[tau - 1] ** 2 for tau in range(1, t + 1))
        np.testing.assert_allclose(v, expect_v, rtol=1e-13)
        vhat = expect_v / (1 - B2 ** t)
        np.testing.assert_allclose(th, th_prev - 1e-3 * U[t - 1] / (np.sqrt(vhat) + EPS), rtol=1e-13)


def test_dense_update_split_numerator_and_scale():
    r = _rng(29)
    P = 50
    th, g, h = r.standard_normal(P), r.standard_normal(P), r.standard_normal(P)
    v0 = np.abs(r.standard_normal(P))
    a = oracle.update_dense(th, v0, g, h=h, lam=0.3, u_scale=0.7, lr=1e-3, beta2=B2, eps=EPS, t=4)
    b = oracle.update_dense(th, v0, 0.7 * (0.7 * g + 0.3 * h), lr=1e-3, beta2=B2, eps=EPS, t=4)
    np.testing.assert_allclose(a[0], b[0], rtol=1e-14)
    np.testing.assert_allclose(a[1], b[1], rtol=1e-14)


def test_factored_equals_dense_for_rank_one_squares():
    # Adafactor identity: when u^2 is exactly rank one on every block (u_ij^2 = a_i b_j), the factored
    # v_hat equals the dense v_hat, for every step if the pattern persists.
    r = _rng(30)
    br, bc = 8, 8
    rows = 20                      # 3 blocks, the last with 4 rows
    P = rows * bc
    a = np.exp(r.standard_normal(rows))
    bb = np.exp(r.standard_normal(bc))
    sign = np.where(r.random((rows, bc)) < 0.5, -1.0, 1.0)
    th = r.standard_normal(P)
    thd, thf = th.copy(), th.copy()
    v = np.zeros(P)
    Rr, Cc = np.zeros(rows), np.zeros(3 * bc)
    for t in range(1, 5):
        scale = 1.0 + 0.5 * t
        u = (sign * np.sqrt(np.outer(a, bb)) * scale).ravel()
        thd, v = oracle.update_dense(thd, v, u, lr=1e-2, beta2=B2, eps=EPS, t=t, weight_decay=0.1)
        thf, Rr, Cc = oracle.update_factored(thf, Rr, Cc, u, lr=1e-2, beta2=B2, eps=EPS, t=t, block_rows=br,
                                             block_cols=bc, weight_decay=0.1)
        np.testing.assert_allclose(thf, thd, rtol=1e-12, atol=1e-15)


def test_factored_statistics_brute_force_and_ragged_tail():
    r = _rng(31)
    br, bc = 4, 8
    P = 11 * 8 + 5                 # 12 rows, the last one short (5 of 8); 3 blocks
    u = r.standard_normal(P)
    th = r.standard_normal(P)
    Rr0, Cc0 = np.abs(r.standard_normal(12)), np.abs(r.standard_normal(3 * bc))
    t = 3
    thf, Rr, Cc = oracle.update_factored(th, Rr0, Cc0, u, lr=1e-2, beta2=B2, eps=EPS, t=t, block_rows=br,
                                         block_cols=bc)
    U2 = np.zeros((12, bc))
    U2.ravel()[:P] = u * u
    np.testing.assert_allclose(Rr, B2 * Rr0 + (1 - B2) * U2.sum(1), rtol=1e-14)
    kap = U2.reshape(3, br, bc).sum(1).ravel()
    np.testing.assert_allclose(Cc, B2 * Cc0 + (1 - B2) * kap, rtol=1e-14)
    vhat = np.zeros((12, bc))
    for blk in range(3):
        rr = Rr[blk * br:(blk + 1) * br]
        vhat[blk * br:(blk + 1) * br] = np.outer(rr, Cc[blk * bc:(blk + 1) * bc]) / rr.sum() / (1 - B2 ** t)
    expect = th - 1e-2 * u / (np.sqrt(vhat.ravel()[:P]) + EPS)
    np.testing.assert_allclose(thf, expect, rtol=1e-13)


def test_factored_zero_block_keeps_decay_only():
    P = 64
    th = _rng(32).standard_normal(P)
    thf, Rr, Cc = oracle.update_factored(th, np.zeros(8), np.zeros(8), np.zeros(P), lr=1e-2, beta2=B2, eps=EPS,
                                         t=1, block_rows=8, block_cols=8, weight_decay=0.1)
    np.testing.assert_allclose(thf, (1 - 1e-3) * th, rtol=1e-15)


# AdamW, the comparison arm of the cost model (appendix "First-order cost accounting"): the dense first
# moment m that BOM deletes, with the same second moment and step map (Sec. 3.5).
def test_adamw_first_step_closed_form():
    # t = 1 from m = v = 0: m_hat = g and v_hat = g^2, so theta_1 = (1 - lr wd) theta - lr g / (|g| + eps)
    r = _rng(40)
    P = 900
    th, g = r.standard_normal(P), r.standard_normal(P) * 1e-3
    g[:4] = 0.0
    segs = [(0, 500, 0.01), (500, 100, 0.0)]
    t1, m1, v1 = oracle.update_adamw(th, np.zeros(P), np.zeros(P), g, lr=1e-2, beta1=0.9, beta2=B2, eps=EPS, t=1,
                                     segments=segs, weight_decay=0.1)
    wd = np.r_[np.full(500, 0.01), np.zeros(100), np.full(300, 0.1)]
    np.testing.assert_allclose(t1, (1 - 1e-2 * wd) * th - 1e-2 * g / (np.abs(g) + EPS), rtol=1e-12, atol=1e-16)
    np.testing.assert_allclose(m1, 0.1 * g, rtol=1e-15)
    np.testing.assert_allclose(v1, (1 - B2) * g * g, rtol=1e-15)


def test_adamw_moments_explicit_sums():
    # m_t = sum_tau (1 - b1) b1^(t - tau) g_tau, v_t likewise with g^2; the step uses their bias corrections
    r = _rng(41)
    P, T, b1 = 48, 6, 0.9
    G = r.standard_normal((T, P))
    th, m, v = r.standard_normal(P), np.zeros(P), np.zeros(P)
    for t in range(1, T + 1):
        th_prev = th
        th, m, v = oracle.update_adamw(th, m, v, G[t - 1], lr=1e-3, beta1=b1, beta2=B2, eps=EPS, t=t)
        em = sum((1 - b1) * b1 ** (t - k) * G[k - 1] for k in range(1, t + 1))
        ev = sum((1 - B2) * B2 ** (t - k) * G[k - 1] ** 2 for k in range(1, t + 1))
        np.testing.assert_allclose(m, em, rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(v, ev, rtol=1e-12)
        step = (em / (1 - b1 ** t)) / (np.sqrt(ev / (1 - B2 ** t)) + EPS)
        np.testing.assert_allclose(th, th_prev - 1e-3 * step, rtol=1e-12, atol=1e-15)


def test_adamw_without_first_moment_is_the_bom_update_of_g():
    # beta1 = 0: m_hat = g, so AdamW takes the same step as the BOM update with numerator g (Sec. 3.5's map)
    r = _rng(42)
    P = 300
    th, g, v0 = r.standard_normal(P), r.standard_normal(P) * 1e-3, np.abs(r.standard_normal(P)) * 1e-6
    segs = [(0, 200, 0.01)]
    ta, _, va = oracle.update_adamw(th, r.standard_normal(P), v0, g, lr=1e-2, beta1=0.0, beta2=B2, eps=EPS, t=3,
                                    segments=segs, weight_decay=0.1, u_scale=0.5)
    tb, vb = oracle.update_dense(th, v0, g, lr=1e-2, beta2=B2, eps=EPS, t=3, segments=segs, weight_decay=0.1,
                                 u_scale=0.5)
    np.testing.assert_allclose(ta, tb, rtol=1e-15)
    np.testing.assert_allclose(va, vb, rtol=1e-15)


def test_adamw_factored_reductions():
    r = _rng(43)
    br, bc = 4, 8
    P = 11 * 8 + 5
    th, g = r.standard_normal(P), r.standard_normal(P) * 1e-3
    Rr0, Cc0 = np.abs(r.standard_normal(12)) * 1e-6, np.abs(r.standard_normal(3 * bc)) * 1e-6
    # beta1 = 0: the factored BOM update of g
    ta, _, Ra, Ca = oracle.update_adamw_factored(th, r.standard_normal(P), Rr0, Cc0, g, lr=1e-2, beta1=0.0, beta2=B2,
                                                 eps=EPS, t=2, block_rows=br, block_cols=bc, weight_decay=0.1)
    tb, Rb, Cb = oracle.update_factored(th, Rr0, Cc0, g, lr=1e-2, beta2=B2, eps=EPS, t=2, block_rows=br, block_cols=bc,
                                        weight_decay=0.1)
    np.testing.assert_allclose(ta, tb, rtol=1e-15)
    np.testing.assert_allclose(Ra, Rb, rtol=1e-15)
    np.testing.assert_allclose(Ca, Cb, rtol=1e-15)
    # g^2 exactly rank one on every block: the factored v_hat is the dense one (Adafactor identity), so the
    # whole AdamW trajectory, first moment included, equals the dense AdamW one
    rows = 20
    P2 = rows * 8
    a, bb = np.exp(r.standard_normal(rows)), np.exp(r.standard_normal(8))
    sign = np.where(r.random((rows, 8)) < 0.5, -1.0, 1.0)
    th2 = r.standard_normal(P2)
    thd, thf, md, mf, v = th2.copy(), th2.copy(), np.zeros(P2), np.zeros(P2), np.zeros(P2)
    Rr, Cc = np.zeros(rows), np.zeros(3 * 8)
    for t in range(1, 5):
        gg = (sign * np.sqrt(np.outer(a, bb)) * (1.0 + 0.5 * t)).ravel()
        thd, md, v = oracle.update_adamw(thd, md, v, gg, lr=1e-2, beta1=0.9, beta2=B2, eps=EPS, t=t, weight_decay=0.1)
        thf, mf, Rr, Cc = oracle.update_adamw_factored(thf, mf, Rr, Cc, gg, lr=1e-2, beta1=0.9, beta2=B2, eps=EPS,
                                                       t=t, block_rows=8, block_cols=8, weight_decay=0.1)
        np.testing.assert_allclose(thf, thd, rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(mf, md, rtol=1e-15)


# Block-shared second moment: Adam-mini's map with the BOM numerator (Sec. 3.5, the substitution into a
# base optimizer's update map; Adam-mini shares one second-moment value per block).
def test_blocks_of_one_are_the_dense_update():
    r = _rng(33)
    P = 700
    th, u, v0 = r.standard_normal(P), r.standard_normal(P) * 1e-3, np.abs(r.standard_normal(P)) * 1e-6
    segs = [(0, 300, 0.01), (300, 150, 0.0), (450, 250, 0.1)]
    tb, vb = oracle.update_blocks(th, v0, u, lr=1e-2, beta2=B2, eps=EPS, t=3, segments=segs, blocks=[1, 1, 1])
    td, vd = oracle.update_dense(th, v0, u, lr=1e-2, beta2=B2, eps=EPS, t=3, segments=segs, weight_decay=0.5)
    np.testing.assert_allclose(tb, td, rtol=1e-15, atol=1e-18)
    np.testing.assert_allclose(vb, vd, rtol=1e-15)


def test_blocks_first_step_closed_form():
    # t = 1, v = 0: v_hat_b is the block mean of u^2. Blocks [1, 2, 2] (mean 3) and [3, 4] (mean 12.5),
    # then [0, 0] (a zero block keeps only the decay) and the single element [-2].
    u = np.array([1.0, 2.0, 2.0, 3.0, 4.0, 0.0, 0.0, -2.0])
    th = np.array([0.0, 0.0, 0.0, 0.0, 0.0, 1.0, -1.0, 0.5])
    segs = [(0, 5, 0.0), (5, 2, 0.5), (7, 1, 0.0)]
    t1, v1 = oracle.update_blocks(th, np.zeros(4), u, lr=0.1, beta2=B2, eps=EPS, t=1, segments=segs,
                                  blocks=[3, 2, 4])
    r3, r12 = math.sqrt(3.0) + EPS, math.sqrt(12.5) + EPS
    expect = [-0.1 / r3, -0.2 / r3, -0.2 / r3, -0.3 / r12, -0.4 / r12, 0.95, -0.95, 0.5 + 0.2 / (2.0 + EPS)]
    np.testing.assert_allclose(t1, expect, rtol=1e-14)
    np.testing.assert_allclose(v1, (1 - B2) * np.array([3.0, 12.5, 0.0, 4.0]), rtol=1e-14)


def test_blocks_second_moment_explicit_sum_and_ragged_tail():
    r = _rng(34)
    P, T, blk = 23, 5, 5           # blocks of 5, 5, 5, 5, 3
    U = r.standard_normal((T, P))
    th = r.standard_normal(P)
    v = np.zeros(5)
    bidx = np.arange(P) // blk
    for t in range(1, T + 1):
        th_prev = th
        th, v = oracle.update_blocks(th, v, U[t - 1], lr=1e-3, beta2=B2, eps=EPS, t=t, segments=[(0, P, 0.0)],
                                     blocks=[blk])
        means = [np.array([np.mean(U[tau - 1][bidx == b] ** 2) for b in range(5)]) for tau in range(1, t + 1)]
        expect_v = sum((1 - B2) * B2 ** (t - tau) * means[tau - 1] for tau in range(1, t + 1))
        np.testing.assert_allclose(v, expect_v, rtol=1e-13)
        vhat = expect_v[bidx] / (1 - B2 ** t)
        np.testing.assert_allclose(th, th_prev - 1e-3 * U[t - 1] / (np.sqrt(vhat) + EPS), rtol=1e-13)


def test_blocks_invariances():
    # a permutation inside every block permutes the step and leaves v unchanged; with eps = 0 the step
    # does not change when the numerator and the second moment are scaled together (u -> k u, v -> k^2 v)
    r = _rng(35)
    P, blk = 48, 12
    th, u, v0 = r.standard_normal(P), r.standard_normal(P), np.abs(r.standard_normal(4))
    perm = np.concatenate([b * blk + r.permutation(blk) for b in range(4)])
    kw = dict(lr=1e-2, beta2=B2, t=2, segments=[(0, P, 0.1)], blocks=[blk])
    ta, va = oracle.update_blocks(th, v0, u, eps=EPS, **kw)
    tp, vp = oracle.update_blocks(th[perm], v0, u[perm], eps=EPS, **kw)
    np.testing.assert_allclose(tp, ta[perm], rtol=1e-14)
    np.testing.assert_allclose(vp, va, rtol=1e-14)
    t0, _ = oracle.update_blocks(th, v0, u, eps=0.0, **kw)
    tk, vk = oracle.update_blocks(th, 9.0 * v0, 3.0 * u, eps=0.0, **kw)
    np.testing.assert_allclose(tk, t0, rtol=1e-13)
    np.testing.assert_allclose(vk, 9.0 * va, rtol=1e-13)


def test_blocks_split_numerator_and_clipping():
    r = _rng(36)
    P = 40
    th, g, h = r.standard_normal(P), r.standard_normal(P), r.standard_normal(P)
    kw = dict(lr=1e-3, beta2=B2, eps=EPS, t=2, segments=[(0, 25, 0.0), (25, 15, 0.1)], blocks=[10, 4])
    v0 = np.abs(r.standard_normal(oracle.blocks_count(kw["segments"], kw["blocks"])))
    a = oracle.update_blocks(th, v0, g, h=h, lam=0.3, u_scale=0.7, clip_norm=0.5, **kw)
    c = oracle.clip_factor(g, h=h, lam=0.3, u_scale=0.7, clip_norm=0.5)
    assert c < 1.0
    b = oracle.update_blocks(th, v0, c * 0.7 * (0.7 * g + 0.3 * h), **kw)
    np.testing.assert_allclose(a[0], b[0], rtol=1e-14)
    np.testing.assert_allclose(a[1], b[1], rtol=1e-14)


# Global-norm clipping of the numerator (appendix "Pretraining Parameters": clipping at 1.0; appendix
# "Conditional Descent and Stationarity": the numerator supplied to the adaptive update includes it).

def test_clip_factor_constant_vector_closed_form():
    # u = a 1 over P elements: ||u|| = |a| sqrt(P), so c = min(1, clip / (|a| sqrt(P) + 1e-6)).
    P, a = 10_000, -3e-3
    u = np.full(P, a)
    for clip in (0.05, 0.2, 0.3, 1.0):
        expect = min(1.0, clip / (abs(a) * math.sqrt(P) + 1e-6))
        assert abs(oracle.clip_factor(u, clip_norm=clip) - expect) <= 1e-12 * expect   # P summed squares
    # u_scale enters the norm: the scaled numerator is what is clipped
    assert abs(oracle.clip_factor(u, u_scale=4.0, clip_norm=0.1) - 0.1 / (4 * abs(a) * 100 + 1e-6)) <= 1e-12
    assert oracle.clip_factor(u, clip_norm=0.0) == 1.0


def test_clip_factor_matches_library_norm_and_split_numerator():
    r = _rng(33)
    P = 4099
    u, h = r.standard_normal(P), r.standard_normal(P)
    n = np.linalg.norm(0.7 * u)
    assert abs(oracle.clip_factor(u, u_scale=0.7, clip_norm=1.5) - 1.5 / (n + 1e-6)) <= 1e-13
    # split mode: the norm is that of the combined numerator (1 - lam) u + lam h, not of u alone
    lam = 0.25
    nm = np.linalg.norm((1 - lam) * u + lam * h)
    assert abs(oracle.clip_factor(u, h=h, lam=lam, clip_norm=2.0) - 2.0 / (nm + 1e-6)) <= 1e-13
    # a history that cancels the current gradient leaves a zero numerator: nothing to clip
    assert oracle.clip_factor(u, h=-(1 - lam) / lam * u, lam=lam, clip_norm=1e-3) == 1.0


def test_clipped_update_is_update_of_scaled_numerator():
    # Clipping is one global rescale of the numerator, applied before both the second moment and the
    # step: the clipped update equals the unclipped update of c u (dense and factored, with an inactive
    # clip leaving the update unchanged).
    r = _rng(34)
    br, bc = 4, 8
    P = 11 * 8 + 4
    th, u = r.standard_normal(P), r.standard_normal(P) * 1e-2
    v0 = np.abs(r.standard_normal(P)) * 1e-4
    Rr0, Cc0 = np.abs(r.standard_normal(12)) * 1e-3, np.abs(r.standard_normal(3 * bc)) * 1e-3
    segs = [(0, 40, 0.01)]
    c = 0.05 / (np.linalg.norm(u) + 1e-6)
    assert c < 1
    kw = dict(lr=1e-2, beta2=B2, eps=EPS, t=3, segments=segs, weight_decay=0.1)
    a = oracle.update_dense(th, v0, u, clip_norm=0.05, **kw)
    b = oracle.update_dense(th, v0, c * u, **kw)
    np.testing.assert_allclose(a[0], b[0], rtol=1e-13)
    np.testing.assert_allclose(a[1], b[1], rtol=1e-12)
    fa = oracle.update_factored(th, Rr0, Cc0, u, block_rows=br, block_cols=bc, clip_norm=0.05, **kw)
    fb = oracle.update_factored(th, Rr0, Cc0, c * u, block_rows=br, block_cols=bc, **kw)
    for x, y in zip(fa, fb):
        np.testing.assert_allclose(x, y, rtol=1e-12)
    big = 10 * np.linalg.norm(u)
    for x, y in zip(oracle.update_dense(th, v0, u, clip_norm=big, **kw), oracle.update_dense(th, v0, u, **kw)):
        np.testing.assert_array_equal(x, y)


# bf16 state storage (appendix "NLP Fine-Tuning Parameters": bf16 parameters and optimizer state).

def test_round_bf16_matches_library_conversion_and_ties():
    import torch
    r = _rng(35)
    x = np.concatenate([r.standard_normal(20000) * 10.0 ** r.integers(-30, 30, 20000),
                        [0.0, -0.0, 1.0, -2.5, 3e38, 1e-39, 2.0 ** -130]]).astype(np.float32)
    lib = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(oracle.round_bf16(x.astype(np.float64)), lib)
    # ties go to the even neighbour; exactly representable values and subnormals stay; below half the
    # smallest subnormal spacing (2^-133) a tie rounds to zero
    cases = {1 + 2.0 ** -8: 0x3F80, 1 + 3 * 2.0 ** -8: 0x3F82, -(1 + 2.0 ** -8): 0xBF80, 0.5: 0x3F00,
             2.0 ** -130: 0x0008, 2.0 ** -134: 0x0000, 3 * 2.0 ** -134: 0x0002}
    got = oracle.round_bf16(np.array(list(cases)))
    np.testing.assert_array_equal(got, np.array(list(cases.values()), np.uint16))
    # the fp64 value is rounded once: a value just above a tie rounds up although its fp32 image is the tie
    assert oracle.round_bf16(np.array([1 + 2.0 ** -8 + 2.0 ** -40]))[0] == 0x3F81


def test_bf16_update_first_step_closed_form():
    # t = 1 on bf16 storage: v_1 = bf16((1 - beta2) u^2), theta_1 = bf16((1 - lr wd) theta - lr u / (|u| + eps)),
    # with theta and u the exact images of their bf16 patterns.
    r = _rng(36)
    P = 3000
    tb = oracle.round_bf16(r.standard_normal(P) * 0.02)
    ub = oracle.round_bf16(r.standard_normal(P) * 1e-3)
    th, u = oracle.bf16_bits_to_f64(tb), oracle.bf16_bits_to_f64(ub)
    t1, v1 = oracle.update_dense_bf16(tb, np.zeros(P, np.uint16), ub, lr=1e-2, beta2=B2, eps=EPS, t=1,
                                      weight_decay=0.05)
    np.testing.assert_array_equal(v1, oracle.round_bf16((1 - B2) * u * u))
    np.testing.assert_array_equal(t1, oracle.round_bf16((1 - 1e-2 * 0.05) * th - 1e-2 * u / (np.abs(u) + EPS)))


# Historical-projection drift telemetry (Sec. 3.3, Eq. (8); appendix "Measuring historical projection drift").

def _tele_batch(r, N, d, V):
    H = r.standard_normal((N, d))
    Z = r.standard_normal((N, V)) * 0.7
    y = r.integers(0, V, N).astype(np.int32)
    y[::4] = -100                       # ignored rows: outside hbar and the cancellation mean
    o = oracle.residual(Z, y)
    return H, y, o


def test_telemetry_fixed_features_have_no_drift():
    # A linear head with the same inputs H at every step has a constant Jacobian, so the own-step EMA of
    # hbar s_t^T equals hbar q_hat_t^T (BOM's reprojection) for any residual sequence: cos 1, drift 0.
    r = _rng(37)
    N, d, V = 12, 5, 7
    H = r.standard_normal((N, d))
    MW, Mb, q = np.zeros((d, V)), np.zeros(V), np.zeros(V)
    for t in range(1, 6):
        Z = r.standard_normal((N, V))
        y = r.integers(0, V, N).astype(np.int32)
        o = oracle.residual(Z, y)
        q, qh = oracle.ema(q, o["s"], B1, t)
        MW, Mb, st = oracle.head_telemetry(H, o["R"], y, o["s"], qh, o["n_valid"], MW, Mb, beta1=B1, t=t)
        assert abs(st["cos"] - 1.0) <= 1e-12 and st["drift"] <= 1e-12
        np.testing.assert_allclose(MW / (1 - B1 ** t), np.outer(H.mean(0), qh), rtol=1e-11, atol=1e-15)


def test_telemetry_explicit_sum_and_moving_features():
    # Changing inputs: Mhat_t is the bias-corrected explicit sum of the own-step projections
    # (1 - beta1) beta1^(t - tau) hbar_tau s_tau^T, and the reported statistics are its cosine and relative
    # distance to hbar_t q_hat_t^T (with the bias part s_tau / q_hat_t), recomputed here with numpy.
    r = _rng(38)
    N, d, V, T = 9, 4, 6, 5
    MW, Mb, q = np.zeros((d, V)), np.zeros(V), np.zeros(V)
    hist = []
    for t in range(1, T + 1):
        H, y, o = _tele_batch(r, N, d, V)
        q, qh = oracle.ema(q, o["s"], B1, t)
        MW, Mb, st = oracle.head_telemetry(H, o["R"], y, o["s"], qh, o["n_valid"], MW, Mb, beta1=B1, t=t)
        hbar = H[y >= 0].mean(0)
        hist.append((hbar, o["s"]))
        bc = 1 - B1 ** t
        MWh = sum((1 - B1) * B1 ** (t - k) * np.outer(hb, sk) for k, (hb, sk) in enumerate(hist, 1)) / bc
        Mbh = sum((1 - B1) * B1 ** (t - k) * sk for k, (_, sk) in enumerate(hist, 1)) / bc
        m = np.concatenate([MWh.ravel(), Mbh])
        h = np.concatenate([np.outer(hbar, qh).ravel(), qh])
        rn = np.linalg.norm(o["R"][y >= 0], axis=1).mean()
        assert abs(st["cancellation"] - np.linalg.norm(o["s"]) / rn) <= 1e-12
        np.testing.assert_allclose(MW / bc, MWh, rtol=1e-12, atol=1e-15)
        assert abs(st["cos"] - m @ h / np.linalg.norm(m) / np.linalg.norm(h)) <= 1e-12
        assert abs(st["drift"] - np.linalg.norm(m - h) / np.linalg.norm(m)) <= 1e-12
        assert abs(st["m_norm"] - np.linalg.norm(m)) <= 1e-12 * np.linalg.norm(m)
    assert st["drift"] > 0.05           # moving features do drift


def test_telemetry_cancellation_ratio():
    # V = 2, equal logits: labels 0 and 1 give r = (-1/2, 1/2) and (1/2, -1/2); they cancel (ratio 0).
    # One supervised row (the other ignored) keeps all of its magnitude (ratio 1).
    H = np.ones((2, 3))
    Z = np.zeros((2, 2))
    for y, expect in (([0, 1], 0.0), ([1, -100], 1.0)):
        y = np.array(y, np.int32)
        o = oracle.residual(Z, y)
        _, _, st = oracle.head_telemetry(H, o["R"], y, o["s"], o["s"], o["n_valid"], np.zeros((3, 2)), beta1=B1, t=1)
        assert abs(st["cancellation"] - expect) <= 1e-15


def test_head_forward_matches_library_matmul():
    # the linear head z_i = W^T h_i + b, against numpy's matrix product (a library routine)
    r = _rng(39)
    H, W, b = r.standard_normal((7, 5)), r.standard_normal((5, 9)), r.standard_normal(9)
    np.testing.assert_allclose(oracle.head_forward(H, W, b), H @ W + b, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(oracle.head_forward(H, W), H @ W, rtol=1e-13, atol=1e-13)


# ----------------------------------------------------------------------------- multi-step

def test_linear_model_bom_equals_own_step_control():
    # Historical-projection appendix: for a linear model on a fixed batch the Jacobian is constant, so
    # BOM's current reprojection and the own-step parameter-space EMA M_t coincide over a trajectory.
    r = _rng(33)
    N, d, V = 32, 6, 5
    H = r.standard_normal((N, d))
    y = r.integers(0, V, N).astype(np.int32)
    theta0 = r.standard_normal(d * V + V) * 0.05
    segs = [(0, d * V, 0.01), (d * V, V, 0.0)]
    kw = dict(d=d, V=V, lr=1e-2, lam=LAM, beta1=B1, beta2=B2, eps=EPS, segments=segs)
    th, v, q = theta0.copy(), np.zeros_like(theta0), np.zeros(V)
    # independent control path: textbook CE gradient + parameter-space EMA of the own-step projection
    th2, v2, M = theta0.copy(), np.zeros_like(theta0), np.zeros_like(theta0)
    wd = np.r_[np.full(d * V, 0.01), np.zeros(V)]
    for t in range(1, 21):
        st = oracle.bom_step_linear_head(H, y, th, v, q, t, **kw)
        th, v, q = st["theta"], st["v"], st["q"]
        W2, b2 = th2[: d * V].reshape(d, V), th2[d * V:]
        P = softmax(H @ W2 + b2, axis=1)
        Rm = P - np.eye(V)[y]
        s = Rm.mean(0)
        g = np.r_[(H.T @ Rm / N).ravel(), s]
        proj = np.r_[np.outer(H.mean(0), s).ravel(), s]     # Jbar_t^T s_t for (W, b)
        M = B1 * M + (1 - B1) * proj
        u2 = (1 - LAM) * g + LAM * M / (1 - B1 ** t)
        v2 = B2 * v2 + (1 - B2) * u2 * u2
        th2 = (1 - 1e-2 * wd) * th2 - 1e-2 * u2 / (np.sqrt(v2 / (1 - B2 ** t)) + EPS)
        np.testing.assert_allclose(st["u"], u2, rtol=1e-9, atol=1e-14)
        np.testing.assert_allclose(th, th2, rtol=1e-9, atol=1e-14)


# ----------------------------------------------------------------------------- accounting

def test_state_accounting_matches_printed_sizes():
    gold = read_golden("state_accounting.txt")
    P = int(gold["p_1b"])
    gib = 2.0 ** 30
    adamw = 4 * P + oracle.state_bytes(P, 32768, "adamw")
    bom = 4 * P + oracle.state_bytes(P, 0, "bom")
    assert round(adamw / gib, 2) == gold["adamw_ckpt_gib_1b"]
    assert round(bom / gib, 2) == gold["bom_ckpt_gib_1b"]
    P4, V4 = int(gold["p_4b"]), int(gold["v_4b"])
    saving = oracle.state_bytes(P4, V4, "adamw") - oracle.state_bytes(P4, V4, "bom")
    assert round(saving / gib, 3) == gold["saving_gib_4b"]


@pytest.mark.parametrize("bad", ["adam", ""])
def test_state_bytes_rejects_unknown(bad):
    with pytest.raises(ValueError):
        oracle.state_bytes(10, 2, bad)


def test_sliced_head_products_equal_full():
    # the wide-output entry points take slices of Z; on the same inputs they equal the full versions
    H, W, b, y = _head_problem(N=40, d=6, V=23, seed=34)
    y[5] = -100
    Z = H @ W + b
    res = oracle.residual(Z, y)
    qh = _rng(35).standard_normal(23) * 0.1
    cols = np.array([0, 3, 22, 7])
    rows = np.array([1, 5, 39])
    full_w = oracle.dW_cols(H, Z, y, res["row_lse"], qh, res["n_valid"], LAM, cols=cols)
    sub_w = oracle.dW_cols_sub(H, Z[:, cols], cols, 23, y, res["row_lse"], qh, res["n_valid"], LAM)
    assert np.array_equal(full_w, sub_w)
    full_h = oracle.dH_rows(W, Z, y, res["row_lse"], qh, res["n_valid"], LAM, rows=rows)
    sub_h = oracle.dH_rows_sub(W, Z[rows], rows, y, res["row_lse"], qh, res["n_valid"], LAM)
    assert np.array_equal(full_h, sub_h)
