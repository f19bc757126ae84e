/*
 * bom_oracle.c -- plain fp64 CPU oracle for one step of Backpropagated Output
 * Momentum (BOM) with AdamW-style scaling.
 *
 * TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this file. It shares no code, header or
 * constant with the GPU library, and the GPU library never calls it.
 *
 * What it follows (paper: "Backpropagated Output Momentum: Relocating
 * Optimizer History from Parameters to Task Space"):
 *   - Algorithm 1 (BOM with AdamW-style scaling): the full step.
 *   - Sec. 3.2 (formal update): residual r = softmax(z) - onehot(y), its batch
 *     mean s, the EMA q and its bias correction q_hat, the mixed objective
 *     (Eq. 3) and its gradient u = (1-lambda) g + lambda Jbar^T q_hat (Eq. 4).
 *   - Appendix "Model and token-level update": the mean runs over the valid
 *     target positions only; ignored targets are excluded from both means.
 *   - Sec. 3.4 (adaptive scaling): v = beta2 v + (1-beta2) u^2,
 *     v_hat = v / (1 - beta2^t), decoupled decay, eps outside the root.
 *
 * All arithmetic is fp64 on the exact fp64 images of the inputs. Loops are
 * plain; the only parallelism is across independent rows, columns or elements
 * (each sum below is still taken in the order its definition writes it).
 *
 * Readings where the paper is silent (each also listed in the design notes):
 *   - a label outside [0, V) that is not ignore_index marks the row invalid
 *     and raises ORC_FLAG_LABEL_RANGE;
 *   - N_t = 0 raises ORC_FLAG_EMPTY and makes s, loss and every gradient 0;
 *   - argmax ties resolve to the lowest index;
 *   - row statistics (lse, argmax) are reported for every row, the label
 *     logit and residual rows only for valid rows (zero otherwise);
 *   - factored second moment (not in the paper): the Adafactor rank-1
 *     factorisation of the same v over blocks of block_rows x block_cols of
 *     the flat buffer, v_hat_ij = R_i C_j / sum(R) / (1 - beta2^t);
 *   - global-norm clipping (a threshold in the paper's protocols, no formula):
 *     the numerator is scaled by min(1, clip / (||u'|| + 1e-6)) over the whole
 *     flat buffer, as PyTorch's clip_grad_norm_ does;
 *   - bf16 state storage: the step is computed on the exact images of the
 *     bf16 inputs and theta and v are rounded once to bf16 (nearest, ties to
 *     even) when stored.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_FLAG_LABEL_RANGE 1
#define ORC_FLAG_EMPTY 2

/* Valid-output set I_t (Algorithm 1; token-level appendix). Returns 1 when row
 * label y is supervised; sets *bad when y is neither ignored nor in range. */
static int orc_is_valid(int32_t y, int64_t V, int32_t ignore_index, int* bad) {
    if (y == ignore_index) return 0;
    if (y < 0 || (int64_t)y >= V) {
        *bad = 1;
        return 0;
    }
    return 1;
}

/*
 * Residual step: Algorithm 1 (the batch-mean residual s_t); Sec. 3.2.
 *   m_i = max_j z_ij, argmax_i = lowest j attaining it, l_i = sum_j exp(z_ij - m_i),
 *   lse_i = m_i + ln l_i; for i in I: r_ij = exp(z_ij - lse_i) - [j = y_i],
 *   CE_i = lse_i - z_{i,y_i}; s_j = (1/N_t) sum_{i in I} r_ij; loss = (1/N_t) sum_{i in I} CE_i.
 * Z is N x V row-major. R (N x V) and the row outputs may be NULL.
 */
void orc_residual(const double* Z, int64_t N, int64_t V, const int32_t* labels, int32_t ignore_index,
                  double* s, double* row_lse, int32_t* row_argmax, double* row_target, double* R,
                  double* loss, int32_t* n_valid, int32_t* flags) {
    int bad = 0;
    int64_t nt = 0;
    char* valid = (char*)malloc((size_t)(N > 0 ? N : 1));
    double* lse = (double*)malloc((size_t)(N > 0 ? N : 1) * sizeof(double));
    for (int64_t i = 0; i < N; ++i) {
        valid[i] = (char)orc_is_valid(labels[i], V, ignore_index, &bad);
        nt += valid[i];
    }

#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < N; ++i) {
        const double* z = Z + i * V;
        double m = z[0];
        int64_t am = 0;
        for (int64_t j = 1; j < V; ++j)
            if (z[j] > m) { m = z[j]; am = j; }
        double l = 0.0;
        for (int64_t j = 0; j < V; ++j) l += exp(z[j] - m);
        lse[i] = m + log(l);
        if (row_lse) row_lse[i] = lse[i];
        if (row_argmax) row_argmax[i] = (int32_t)am;
        if (row_target) row_target[i] = valid[i] ? z[labels[i]] : 0.0;
        if (R) {
            double* r = R + i * V;
            for (int64_t j = 0; j < V; ++j)
                r[j] = valid[i] ? exp(z[j] - lse[i]) - (j == labels[i] ? 1.0 : 0.0) : 0.0;
        }
    }

    /* s_j: a sum over the valid rows in row order, one column at a time. */
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < V; ++j) {
        double acc = 0.0;
        for (int64_t i = 0; i < N; ++i)
            if (valid[i]) acc += exp(Z[i * V + j] - lse[i]) - (j == labels[i] ? 1.0 : 0.0);
        s[j] = nt > 0 ? acc / (double)nt : 0.0;
    }

    double ce = 0.0;
    for (int64_t i = 0; i < N; ++i)
        if (valid[i]) ce += lse[i] - Z[i * V + labels[i]];
    *loss = nt > 0 ? ce / (double)nt : 0.0;
    *n_valid = (int32_t)nt;
    *flags = (bad ? ORC_FLAG_LABEL_RANGE : 0) | (nt == 0 ? ORC_FLAG_EMPTY : 0);
    free(valid);
    free(lse);
}

/*
 * Task-space EMA: Sec. 3.2 and Algorithm 1:
 *   q_t = beta1 q_{t-1} + (1 - beta1) s_t,  q_hat_t = q_t / (1 - beta1^t),  t >= 1.
 */
void orc_ema(double* q, const double* s, int64_t V, double beta1, int64_t t, double* q_hat) {
    double bc = 1.0 - pow(beta1, (double)t);
    for (int64_t j = 0; j < V; ++j) {
        q[j] = beta1 * q[j] + (1.0 - beta1) * s[j];
        q_hat[j] = q[j] / bc;
    }
}

/*
 * Gradient of the mixed objective (Eq. 3) with respect to logit z_ij, with q_hat
 * held constant: G_ij = [i in I] ((1 - lambda) r_ij + lambda q_hat_j) / N_t.
 */
static double orc_g(const double* Z, int64_t V, int64_t i, int64_t j, const int32_t* labels,
                    int32_t ignore_index, const double* row_lse, const double* q_hat, int64_t n_valid,
                    double lambda) {
    int bad = 0;
    if (n_valid <= 0 || !orc_is_valid(labels[i], V, ignore_index, &bad)) return 0.0;
    double r = exp(Z[i * V + j] - row_lse[i]) - (j == labels[i] ? 1.0 : 0.0);
    return ((1.0 - lambda) * r + lambda * q_hat[j]) / (double)n_valid;
}

/*
 * Head weight gradient, selected columns: for the linear head z_i = W^T h_i (+ b),
 * dL_mix/dW = H^T G, so column j of dW is sum_i H_i G_ij (Eq. 4, head block).
 * H is N x d, Z is N x V; out is d x ncols (row-major).
 */
void orc_dW_cols(const double* H, int64_t N, int64_t d, const double* Z, int64_t V, const int32_t* labels,
                 int32_t ignore_index, const double* row_lse, const double* q_hat, int64_t n_valid,
                 double lambda, const int64_t* cols, int64_t ncols, double* out) {
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t c = 0; c < ncols; ++c) {
        int64_t j = cols[c];
        double* g = (double*)malloc((size_t)(N > 0 ? N : 1) * sizeof(double));
        for (int64_t i = 0; i < N; ++i) g[i] = orc_g(Z, V, i, j, labels, ignore_index, row_lse, q_hat, n_valid, lambda);
        for (int64_t k = 0; k < d; ++k) {
            double acc = 0.0;
            for (int64_t i = 0; i < N; ++i) acc += H[i * d + k] * g[i];
            out[k * ncols + c] = acc;
        }
        free(g);
    }
}

/*
 * Head input gradient, selected rows: dL_mix/dH = G W^T, so row i of dH is
 * sum_j G_ij W[:, j]. W is d x V (row-major); out is nrows x d.
 */
void orc_dH_rows(const double* W, int64_t d, const double* Z, int64_t V, const int32_t* labels,
                 int32_t ignore_index, const double* row_lse, const double* q_hat, int64_t n_valid,
                 double lambda, const int64_t* rows, int64_t nrows, double* out) {
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t c = 0; c < nrows; ++c) {
        int64_t i = rows[c];
        double* g = (double*)malloc((size_t)(V > 0 ? V : 1) * sizeof(double));
        for (int64_t j = 0; j < V; ++j) g[j] = orc_g(Z, V, i, j, labels, ignore_index, row_lse, q_hat, n_valid, lambda);
        for (int64_t k = 0; k < d; ++k) {
            double acc = 0.0;
            for (int64_t j = 0; j < V; ++j) acc += g[j] * W[k * V + j];
            out[c * d + k] = acc;
        }
        free(g);
    }
}

/*
 * The same head products for very wide outputs, from slices of Z: Zc holds the columns cols[0..ncols)
 * of Z (N x ncols, row-major) for dW; Zr holds the rows rows[0..nrows) of Z (nrows x V) for dH.
 * G_ij is the same definition as orc_g.
 */
static double orc_g_val(double z, int64_t V, int64_t j, int32_t y, int32_t ignore_index, double lse, double qh,
                        int64_t n_valid, double lambda) {
    int bad = 0;
    if (n_valid <= 0 || !orc_is_valid(y, V, ignore_index, &bad)) return 0.0;
    double r = exp(z - lse) - (j == y ? 1.0 : 0.0);
    return ((1.0 - lambda) * r + lambda * qh) / (double)n_valid;
}

void orc_dW_cols_sub(const double* H, int64_t N, int64_t d, const double* Zc, int64_t V, const int32_t* labels,
                     int32_t ignore_index, const double* row_lse, const double* q_hat, int64_t n_valid, double lambda,
                     const int64_t* cols, int64_t ncols, double* out) {
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t c = 0; c < ncols; ++c) {
        int64_t j = cols[c];
        double* g = (double*)malloc((size_t)(N > 0 ? N : 1) * sizeof(double));
        for (int64_t i = 0; i < N; ++i)
            g[i] = orc_g_val(Zc[i * ncols + c], V, j, labels[i], ignore_index, row_lse[i], q_hat[j], n_valid, lambda);
        for (int64_t k = 0; k < d; ++k) {
            double acc = 0.0;
            for (int64_t i = 0; i < N; ++i) acc += H[i * d + k] * g[i];
            out[k * ncols + c] = acc;
        }
        free(g);
    }
}

void orc_dH_rows_sub(const double* W, int64_t d, const double* Zr, int64_t V, const int32_t* labels,
                     int32_t ignore_index, const double* row_lse, const double* q_hat, int64_t n_valid, double lambda,
                     const int64_t* rows, int64_t nrows, double* out) {
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t c = 0; c < nrows; ++c) {
        int64_t i = rows[c];
        double* g = (double*)malloc((size_t)(V > 0 ? V : 1) * sizeof(double));
        for (int64_t j = 0; j < V; ++j)
            g[j] = orc_g_val(Zr[c * V + j], V, j, labels[i], ignore_index, row_lse[i], q_hat[j], n_valid, lambda);
        for (int64_t k = 0; k < d; ++k) {
            double acc = 0.0;
            for (int64_t j = 0; j < V; ++j) acc += g[j] * W[k * V + j];
            out[c * d + k] = acc;
        }
        free(g);
    }
}

/* Head bias gradient: the bias Jacobian is the identity, so db_j = sum_i G_ij. */
void orc_db(const double* Z, int64_t N, int64_t V, const int32_t* labels, int32_t ignore_index,
            const double* row_lse, const double* q_hat, int64_t n_valid, double lambda, double* db) {
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < V; ++j) {
        double acc = 0.0;
        for (int64_t i = 0; i < N; ++i) acc += orc_g(Z, V, i, j, labels, ignore_index, row_lse, q_hat, n_valid, lambda);
        db[j] = acc;
    }
}

/* Decoupled weight decay of flat element e: the segment that covers e, else wd_default. */
static double orc_decay_of(int64_t e, const int64_t* seg_off, const int64_t* seg_len, const double* seg_wd,
                           int nsegs, double wd_default) {
    for (int k = 0; k < nsegs; ++k)
        if (e >= seg_off[k] && e < seg_off[k] + seg_len[k]) return seg_wd[k];
    return wd_default;
}

/* Update numerator: u' = u_scale * u, or in split mode u' = u_scale * ((1 - lambda) u + lambda h). */
static double orc_numerator(const double* u, const double* h, int64_t e, double lambda, double u_scale) {
    if (h) return u_scale * ((1.0 - lambda) * u[e] + lambda * h[e]);
    return u_scale * u[e];
}

/*
 * Global-norm clipping of the update numerator (appendix "Pretraining Parameters" and appendix
 * "Memory and Timing Protocols": clipping at 1.0; appendix "Conditional Descent and Stationarity":
 * the numerator supplied to the adaptive update includes the clipping). Returns the factor
 *   c = min(1, clip_norm / (||u'|| + 1e-6)),
 * ||u'|| the L2 norm of the numerator of orc_numerator over all P elements (summed in element
 * order). The clipped numerator c u' then enters both the second moment and the parameter step.
 * The 1e-6 guard is a reading (PyTorch's clip_grad_norm_); the paper gives only the threshold.
 */
double orc_clip_factor(const double* u, const double* h, int64_t P, double lambda, double u_scale, double clip_norm) {
    double ss = 0.0;
    for (int64_t e = 0; e < P; ++e) {
        double up = orc_numerator(u, h, e, lambda, u_scale);
        ss += up * up;
    }
    double c = clip_norm / (sqrt(ss) + 1e-6);
    return c < 1.0 ? c : 1.0;
}

/*
 * Dense second moment and parameter update: Sec. 3.4 and Algorithm 1:
 *   v = beta2 v + (1 - beta2) u'^2; v_hat = v / (1 - beta2^t);
 *   theta = (1 - lr * omega) theta - lr * u' / (sqrt(v_hat) + eps).
 */
void orc_update_dense(double* theta, double* v, const double* u, const double* h, int64_t P,
                      const int64_t* seg_off, const int64_t* seg_len, const double* seg_wd, int nsegs,
                      double wd_default, double lr, double beta2, double eps, double lambda, double u_scale,
                      int64_t t) {
    double bc2 = 1.0 - pow(beta2, (double)t);
#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < P; ++e) {
        double up = orc_numerator(u, h, e, lambda, u_scale);
        double om = orc_decay_of(e, seg_off, seg_len, seg_wd, nsegs, wd_default);
        v[e] = beta2 * v[e] + (1.0 - beta2) * up * up;
        double vhat = v[e] / bc2;
        theta[e] = (1.0 - lr * om) * theta[e] - lr * up / (sqrt(vhat) + eps);
    }
}

/*
 * Factored second moment (Adafactor-style rank-1 factorisation of the same v).
 * The flat buffer is a row-major matrix with block_cols columns (the last row
 * may be short); consecutive groups of block_rows rows form a block. Per block:
 *   rho_i = sum_j u'_ij^2, kappa_j = sum_i u'_ij^2 (over the elements present);
 *   Rr_i = beta2 Rr_i + (1 - beta2) rho_i;  Cc_j = beta2 Cc_j + (1 - beta2) kappa_j;
 *   v_hat_ij = Rr_i Cc_j / (sum_{k in block} Rr_k) / (1 - beta2^t)  (0 when that sum is 0);
 *   theta_ij = (1 - lr * omega) theta_ij - lr * u'_ij / (sqrt(v_hat_ij) + eps).
 * Rr has one entry per row (ceil(P / block_cols)); Cc has block_cols entries per block.
 */
void orc_update_factored(double* theta, double* Rr, double* Cc, const double* u, const double* h, int64_t P,
                         int64_t block_rows, int64_t block_cols, const int64_t* seg_off, const int64_t* seg_len,
                         const double* seg_wd, int nsegs, double wd_default, double lr, double beta2, double eps,
                         double lambda, double u_scale, int64_t t) {
    double bc2 = 1.0 - pow(beta2, (double)t);
    int64_t nrows = (P + block_cols - 1) / block_cols;
    int64_t nblocks = (nrows + block_rows - 1) / block_rows;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < nblocks; ++b) {
        int64_t r0 = b * block_rows;
        int64_t r1 = r0 + block_rows < nrows ? r0 + block_rows : nrows;
        double* kappa = (double*)calloc((size_t)block_cols, sizeof(double));
        double* Cb = Cc + b * block_cols;
        for (int64_t i = r0; i < r1; ++i) {
            double rho = 0.0;
            for (int64_t j = 0; j < block_cols; ++j) {
                int64_t e = i * block_cols + j;
                if (e >= P) break;
                double up = orc_numerator(u, h, e, lambda, u_scale);
                rho += up * up;
                kappa[j] += up * up;
            }
            Rr[i] = beta2 * Rr[i] + (1.0 - beta2) * rho;
        }
        for (int64_t j = 0; j < block_cols; ++j) Cb[j] = beta2 * Cb[j] + (1.0 - beta2) * kappa[j];
        double rsum = 0.0;
        for (int64_t i = r0; i < r1; ++i) rsum += Rr[i];
        for (int64_t i = r0; i < r1; ++i) {
            for (int64_t j = 0; j < block_cols; ++j) {
                int64_t e = i * block_cols + j;
                if (e >= P) break;
                double up = orc_numerator(u, h, e, lambda, u_scale);
                double om = orc_decay_of(e, seg_off, seg_len, seg_wd, nsegs, wd_default);
                double vhat = rsum > 0.0 ? Rr[i] * Cb[j] / rsum / bc2 : 0.0;
                theta[e] = (1.0 - lr * om) * theta[e] - lr * up / (sqrt(vhat) + eps);
            }
        }
        free(kappa);
    }
}

/*
 * AdamW, the comparison optimizer whose dense first moment BOM deletes (Sec. 1: an EMA m_t of the
 * gradients beside every tensor; Sec. 3.5: its update map a / (sqrt(v_hat) + eps) applied to the
 * bias-corrected first moment m_hat = m / (1 - beta1^t)). It is here as the other arm of the cost model of
 * appendix "First-order cost accounting" (Delta t = alpha N_out - beta P: deleting m removes its
 * maintenance over the P elements). With g the gradient (times u_scale):
 *   m = beta1 m + (1 - beta1) g;  v = beta2 v + (1 - beta2) g^2;
 *   theta = (1 - lr * omega) theta - lr * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps).
 */
void orc_update_adamw(double* theta, double* m, double* v, const double* g, int64_t P, const int64_t* seg_off,
                      const int64_t* seg_len, const double* seg_wd, int nsegs, double wd_default, double lr,
                      double beta1, double beta2, double eps, double u_scale, int64_t t) {
    double bc1 = 1.0 - pow(beta1, (double)t);
    double bc2 = 1.0 - pow(beta2, (double)t);
#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < P; ++e) {
        double ge = u_scale * g[e];
        double om = orc_decay_of(e, seg_off, seg_len, seg_wd, nsegs, wd_default);
        m[e] = beta1 * m[e] + (1.0 - beta1) * ge;
        v[e] = beta2 * v[e] + (1.0 - beta2) * ge * ge;
        double mhat = m[e] / bc1;
        double vhat = v[e] / bc2;
        theta[e] = (1.0 - lr * om) * theta[e] - lr * mhat / (sqrt(vhat) + eps);
    }
}

/*
 * AdamW with the factored second moment of orc_update_factored (the same reading, here of g^2): the dense
 * first moment m as in orc_update_adamw, v_hat_ij = Rr_i Cc_j / (sum_{k in block} Rr_k) / (1 - beta2^t).
 */
void orc_update_adamw_factored(double* theta, double* m, double* Rr, double* Cc, const double* g, int64_t P,
                               int64_t block_rows, int64_t block_cols, const int64_t* seg_off, const int64_t* seg_len,
                               const double* seg_wd, int nsegs, double wd_default, double lr, double beta1,
                               double beta2, double eps, double u_scale, int64_t t) {
    double bc1 = 1.0 - pow(beta1, (double)t);
    double bc2 = 1.0 - pow(beta2, (double)t);
    int64_t nrows = (P + block_cols - 1) / block_cols;
    int64_t nblocks = (nrows + block_rows - 1) / block_rows;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < nblocks; ++b) {
        int64_t r0 = b * block_rows;
        int64_t r1 = r0 + block_rows < nrows ? r0 + block_rows : nrows;
        double* kappa = (double*)calloc((size_t)block_cols, sizeof(double));
        double* Cb = Cc + b * block_cols;
        for (int64_t i = r0; i < r1; ++i) {
            double rho = 0.0;
            for (int64_t j = 0; j < block_cols; ++j) {
                int64_t e = i * block_cols + j;
                if (e >= P) break;
                double ge = u_scale * g[e];
                rho += ge * ge;
                kappa[j] += ge * ge;
            }
            Rr[i] = beta2 * Rr[i] + (1.0 - beta2) * rho;
        }
        for (int64_t j = 0; j < block_cols; ++j) Cb[j] = beta2 * Cb[j] + (1.0 - beta2) * kappa[j];
        double rsum = 0.0;
        for (int64_t i = r0; i < r1; ++i) rsum += Rr[i];
        for (int64_t i = r0; i < r1; ++i) {
            for (int64_t j = 0; j < block_cols; ++j) {
                int64_t e = i * block_cols + j;
                if (e >= P) break;
                double ge = u_scale * g[e];
                double om = orc_decay_of(e, seg_off, seg_len, seg_wd, nsegs, wd_default);
                m[e] = beta1 * m[e] + (1.0 - beta1) * ge;
                double vhat = rsum > 0.0 ? Rr[i] * Cb[j] / rsum / bc2 : 0.0;
                theta[e] = (1.0 - lr * om) * theta[e] - lr * (m[e] / bc1) / (sqrt(vhat) + eps);
            }
        }
        free(kappa);
    }
}

/*
 * Block-shared second moment: Adam-mini's update map driven by the BOM numerator. Sec. 3.5 deletes the
 * base optimizer's first moment and feeds the numerator u' to its map Phi(a, v); for Adam-mini that map
 * is a / (sqrt(v_hat) + eps) with one second-moment value per block of parameters, the block average of
 * the squared numerator feeding its EMA. The segments tile [0, P) in order and segment k is cut into
 * consecutive blocks of seg_blk[k] elements (the last one may be shorter). For block b with elements E_b:
 *   v_b = beta2 v_b + (1 - beta2) (1/|E_b|) sum_{e in E_b} u'_e^2,   v_hat_b = v_b / (1 - beta2^t),
 *   theta_e = (1 - lr * omega_k) theta_e - lr * u'_e / (sqrt(v_hat_b) + eps),
 * omega_k the weight decay of the segment. v lists the blocks of segment 0, then of segment 1, ...
 * A block length of 1 is the elementwise second moment of orc_update_dense.
 */
void orc_update_blocks(double* theta, double* v, const double* u, const double* h, int64_t P,
                       const int64_t* seg_off, const int64_t* seg_len, const double* seg_wd, const int64_t* seg_blk,
                       int nsegs, double lr, double beta2, double eps, double lambda, double u_scale, int64_t t) {
    double bc2 = 1.0 - pow(beta2, (double)t);
    int64_t vbase = 0;
    (void)P;
    for (int k = 0; k < nsegs; ++k) {
        int64_t len = seg_len[k], blk = seg_blk[k];
        int64_t nblk = (len + blk - 1) / blk;
#pragma omp parallel for schedule(static)
        for (int64_t b = 0; b < nblk; ++b) {
            int64_t e0 = seg_off[k] + b * blk;
            int64_t e1 = e0 + blk < seg_off[k] + len ? e0 + blk : seg_off[k] + len;
            double ss = 0.0;
            for (int64_t e = e0; e < e1; ++e) {
                double up = orc_numerator(u, h, e, lambda, u_scale);
                ss += up * up;
            }
            double* vb = v + vbase + b;
            *vb = beta2 * *vb + (1.0 - beta2) * ss / (double)(e1 - e0);
            double denom = sqrt(*vb / bc2) + eps;
            for (int64_t e = e0; e < e1; ++e) {
                double up = orc_numerator(u, h, e, lambda, u_scale);
                theta[e] = (1.0 - lr * seg_wd[k]) * theta[e] - lr * up / denom;
            }
        }
        vbase += nblk;
    }
}

/*
 * Historical-projection drift telemetry of the linear head (Sec. 3.3, Eq. (8);
 * appendix "Historical-Projection Control" and appendix "Measuring historical projection drift").
 * For z_i = W^T h_i + b the batch-mean Jacobian maps a task-space vector x to Jbar^T x = (hbar x^T, x),
 * hbar = (1/N_t) sum_{i in I} H_i. One telemetry step:
 *   M_W = beta1 M_W + (1 - beta1) hbar s^T,   M_b = beta1 M_b + (1 - beta1) s   (own-step projections),
 *   Mhat = M / (1 - beta1^t),   h = (hbar q_hat^T, q_hat)                     (BOM's reprojection),
 *   out[0] = cos(Mhat, h), out[1] = ||Mhat - h|| / ||Mhat||,
 *   out[2] = ||s|| / ((1/N_t) sum_{i in I} ||r_i||)   (within-batch cancellation),
 *   out[3] = ||Mhat||, out[4] = ||h||.
 * The head is W and, when M_b is not NULL, b. R holds the residual rows (rows outside I are zero).
 * N_t = 0 leaves M unchanged by the projections (hbar = 0, s = 0) and reports 0 for the ratios.
 */
void orc_head_telemetry(const double* H, int64_t N, int64_t d, const double* R, int64_t V, const int32_t* labels,
                        int32_t ignore_index, const double* s, const double* q_hat, int64_t n_valid, double* M_W,
                        double* M_b, double beta1, int64_t t, double* out) {
    double* hbar = (double*)calloc((size_t)d, sizeof(double));
    double rnorm_sum = 0.0;
    for (int64_t i = 0; i < N; ++i) {
        int bad = 0;
        if (!orc_is_valid(labels[i], V, ignore_index, &bad)) continue;
        for (int64_t k = 0; k < d; ++k) hbar[k] += H[i * d + k];
        double rr = 0.0;
        for (int64_t j = 0; j < V; ++j) rr += R[i * V + j] * R[i * V + j];
        rnorm_sum += sqrt(rr);
    }
    for (int64_t k = 0; k < d; ++k) hbar[k] = n_valid > 0 ? hbar[k] / (double)n_valid : 0.0;
    double inv_bc = 1.0 / (1.0 - pow(beta1, (double)t));
    double mm = 0.0, mh = 0.0, hh = 0.0, dd = 0.0, ss = 0.0;
    for (int64_t k = 0; k < d; ++k)
        for (int64_t j = 0; j < V; ++j) {
            double* m = &M_W[k * V + j];
            *m = beta1 * *m + (1.0 - beta1) * hbar[k] * s[j];
            double mhat = *m * inv_bc, hv = hbar[k] * q_hat[j];
            mm += mhat * mhat;
            mh += mhat * hv;
            hh += hv * hv;
            dd += (mhat - hv) * (mhat - hv);
        }
    if (M_b)
        for (int64_t j = 0; j < V; ++j) {
            M_b[j] = beta1 * M_b[j] + (1.0 - beta1) * s[j];
            double mhat = M_b[j] * inv_bc, hv = q_hat[j];
            mm += mhat * mhat;
            mh += mhat * hv;
            hh += hv * hv;
            dd += (mhat - hv) * (mhat - hv);
        }
    for (int64_t j = 0; j < V; ++j) ss += s[j] * s[j];
    double rmean = n_valid > 0 ? rnorm_sum / (double)n_valid : 0.0;
    out[0] = mm > 0.0 && hh > 0.0 ? mh / (sqrt(mm) * sqrt(hh)) : 0.0;
    out[1] = mm > 0.0 ? sqrt(dd) / sqrt(mm) : 0.0;
    out[2] = rmean > 0.0 ? sqrt(ss) / rmean : 0.0;
    out[3] = sqrt(mm);
    out[4] = sqrt(hh);
    free(hbar);
}

/*
 * bf16 storage (appendix "NLP Fine-Tuning Parameters": bf16 parameter and optimizer-state storage,
 * the task-space EMA kept in fp32). Rounds each fp64 value once to the nearest bf16 (8 significant
 * bits, ties to even; bf16 has fp32's exponent range, so below 2^-126 the spacing is 2^-133) and
 * returns its bit pattern. The bf16 step is the fp64 step on the exact fp64 images of the bf16
 * inputs, with theta and v rounded this way when they are stored.
 */
void orc_round_bf16(const double* x, int64_t n, uint16_t* out) {
    for (int64_t k = 0; k < n; ++k) {
        double v = x[k], r;
        if (v == 0.0 || !isfinite(v)) {
            r = v;
        } else {
            int e;
            frexp(v, &e);                          /* |v| = m 2^e, 0.5 <= m < 1 */
            int q = e - 8;                         /* spacing of 8 significant bits */
            if (q < -133) q = -133;                /* subnormal bf16 spacing */
            r = ldexp(nearbyint(ldexp(v, -q)), q); /* round half to even (default rounding mode) */
        }
        float f = (float)r;                        /* exact: r has at most 8 significant bits */
        uint32_t bits;
        memcpy(&bits, &f, 4);
        out[k] = (uint16_t)(bits >> 16);
    }
}

/*
 * Linear-head forward used by the multi-step loop: z_i = W^T h_i + b.
 * H is N x d, W is d x V, b has V entries (may be NULL); Z is N x V.
 */
void orc_head_forward(const double* H, int64_t N, int64_t d, const double* W, int64_t V, const double* b,
                      double* Z) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < N; ++i)
        for (int64_t j = 0; j < V; ++j) {
            double acc = b ? b[j] : 0.0;
            for (int64_t k = 0; k < d; ++k) acc += H[i * d + k] * W[k * V + j];
            Z[i * V + j] = acc;
        }
}
