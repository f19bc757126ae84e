/*
 * bom.h -- C-ABI of libbom.so: the per-step hot path of Backpropagated Output
 * Momentum (BOM) with AdamW-style scaling on one AMD Instinct MI355X (gfx950).
 *
 * The method (paper: "Backpropagated Output Momentum: Relocating Optimizer
 * History from Parameters to Task Space", Algorithm 1) keeps one task-space
 * EMA q of the batch-mean softmax-cross-entropy residual s instead of a
 * parameter-shaped first moment, folds its bias-corrected value q_hat into the
 * gradient of the logits, and updates the parameters with a second moment of
 * the resulting numerator u and decoupled weight decay.
 *
 * One step on the hot path is four calls, enqueued in this order:
 *   bom_residual  -> s, row statistics, R           (Algorithm 1: s_t)
 *   bom_ema       -> q (in place), q_hat            (Algorithm 1: q_t, q_hat_t)
 *   bom_head_vjp  -> dW, db, dH of the mixed loss   (Eq. 3 / Eq. 4, output head)
 *   bom_update    -> theta, v in place              (Sec. 3.4; Algorithm 1, the update)
 *
 * Conventions shared by every entry point:
 *   - Every array argument is caller-owned DEVICE memory, except the small
 *     host structs `segs` and `cfg`. The library allocates nothing and keeps
 *     no pointer after returning; buffers must stay alive until the stream
 *     reaches the enqueued work.
 *   - `stream` is a hipStream_t (NULL = the default stream). Every call only
 *     enqueues work; none synchronises the host.
 *   - Matrices are row-major with an explicit leading dimension in ELEMENTS.
 *   - Arguments are validated on the host before anything is enqueued; on an
 *     argument error nothing is launched. bom_last_error() returns a
 *     thread-local description of the last failure. No exception, abort or
 *     exit crosses this ABI.
 *   - Data-dependent conditions are reported in a device `flags` word
 *     (BOM_FLAG_*), never by the return status.
 *   - Results are deterministic: the same inputs give bitwise-identical
 *     outputs (no floating-point atomics; fixed reduction orders).
 */
#ifndef BOM_H
#define BOM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    BOM_OK = 0,
    BOM_ERR_NULL = 1,        /* a required pointer is NULL */
    BOM_ERR_SHAPE = 2,       /* a size or leading dimension is out of range */
    BOM_ERR_DTYPE = 3,       /* an unsupported dtype combination */
    BOM_ERR_HYPER = 4,       /* a hyperparameter is outside its domain */
    BOM_ERR_WORKSPACE = 5,   /* workspace missing or smaller than the query returns */
    BOM_ERR_ALIAS = 6,       /* buffers that must be distinct overlap */
    BOM_ERR_HIP = 7,         /* a HIP runtime call failed (detail in bom_last_error) */
    BOM_ERR_UNSUPPORTED = 8  /* valid request this library does not implement */
} bom_status;

typedef enum { BOM_F32 = 0, BOM_BF16 = 1 } bom_dtype;

/* Bits of the device flags word written by bom_residual. */
#define BOM_FLAG_LABEL_RANGE 1 /* some label was neither ignore_index nor in [0, V); that row is ignored */
#define BOM_FLAG_EMPTY 2       /* no valid row (N_t = 0): s = 0, loss = 0, downstream gradients are 0 */
/* Informational: rows too wide for one workgroup are shared by several workgroups that exchange
 * per-part row records with a bounded wait; a workgroup whose wait ran out recomputed the missing
 * records from Z with the same operations in the same order. Every output is bitwise the same as
 * without it; the bit only tells that the exchange was slow. */
#define BOM_FLAG_RESIDUAL_RECOMPUTED 4

/* Second-moment layouts of bom_update. */
#define BOM_V_DENSE 0
#define BOM_V_FACTORED 1
#define BOM_V_BLOCKS 2

#define BOM_MAX_SEGMENTS 16

/* ------------------------------------------------------------------------------------------
 * bom_residual -- Algorithm 1 (the batch-mean residual s_t); Sec. 3.2 (r = softmax(z) - onehot(y));
 * token-level form: the appendix on language models (each valid target position is an
 * example; ignored targets are excluded from every mean).
 *
 * For every row i of Z [N, V] (leading dimension ldz, dtype z_dt):
 *   m_i = max_j z_ij, row_argmax[i] = the lowest j attaining m_i,
 *   row_lse[i] = m_i + ln sum_j exp(z_ij - m_i).
 * Row i is valid (i in I) when labels[i] != ignore_index and 0 <= labels[i] < V.
 * For valid rows: row_target[i] = z_{i,y_i} (an exact copy of the input element),
 *   R_ij = exp(z_ij - row_lse[i]) - [j == y_i]; for other rows row_target[i] = 0 and R_i = 0.
 * Then, with N_t = |I|:
 *   s[j] = (1/N_t) sum_{i in I} R_ij,   *loss = (1/N_t) sum_{i in I} (row_lse[i] - z_{i,y_i}),
 *   *n_valid = N_t,   *flags = BOM_FLAG_* bits (overwritten, not OR-ed).
 * If N_t = 0: s = 0, *loss = 0 and BOM_FLAG_EMPTY is set.
 *
 *   Z         device [N, ldz] of z_dt (BOM_F32 or BOM_BF16); ldz >= V.
 *   labels    device int32 [N].
 *   s         device fp32 [V].              row_lse device fp32 [N].
 *   row_argmax, row_target: device [N] (int32 / fp32), may be NULL.
 *   R         device [N, ldr] of r_dt, may be NULL (then R is not written). r_dt must equal
 *             z_dt. ldr >= V.
 *   loss      device fp32 [1].  n_valid device int32 [1].  flags device int32 [1].
 *   workspace device, at least bom_residual_workspace_bytes(N, V, z_dt) bytes, 256-byte aligned;
 *             contents on entry are ignored. It holds per-workgroup partial sums and, for rows
 *             too wide for one workgroup, the records the workgroups sharing a row exchange, so
 *             calls that may run at the same time must not share it.
 * Errors: BOM_ERR_NULL, BOM_ERR_SHAPE (N < 1, V < 2, ld < V, N or V >= 2^31), BOM_ERR_DTYPE,
 *         BOM_ERR_WORKSPACE, BOM_ERR_HIP.
 * ---------------------------------------------------------------------------------------- */
size_t bom_residual_workspace_bytes(int64_t N, int64_t V, bom_dtype z_dt);
bom_status bom_residual(const void* Z, bom_dtype z_dt, int64_t N, int64_t V, int64_t ldz,
                        const int32_t* labels, int32_t ignore_index,
                        float* s, float* row_lse, int32_t* row_argmax, float* row_target,
                        void* R, bom_dtype r_dt, int64_t ldr,
                        float* loss, int32_t* n_valid, int32_t* flags,
                        void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------------------------
 * bom_residual_noalloc -- for callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation): bom_residual with the library's own fixed
 * scratch array in place of the workspace. Same arguments, outputs and errors as bom_residual, without
 * workspace and ws_bytes; it allocates nothing (no hipMalloc, no allocating library routine).
 *
 * The scratch is a device array of BOM_RESIDUAL_SCRATCH_BYTES that every device the library runs on holds
 * until the process ends; its address on the current device (the stream must belong to the device that
 * is current) is looked up on the first call on that device. A shape whose workspace would exceed it
 * (bom_residual_workspace_bytes(N, V, z_dt) > BOM_RESIDUAL_SCRATCH_BYTES; e.g. V above about 60,000
 * bf16 columns) returns BOM_ERR_WORKSPACE before anything is enqueued. Every call on one device shares
 * that device's array and leaves its last contents there (each call rewrites what it reads, and clears
 * what must start at zero with a kernel, not a memset), so calls that may overlap on one device (other
 * streams, other threads) race: serialise them, or use bom_residual with separate workspaces.
 * ---------------------------------------------------------------------------------------- */
#define BOM_RESIDUAL_SCRATCH_BYTES ((size_t)64 << 20)
bom_status bom_residual_noalloc(const void* Z, bom_dtype z_dt, int64_t N, int64_t V, int64_t ldz,
                                const int32_t* labels, int32_t ignore_index,
                                float* s, float* row_lse, int32_t* row_argmax, float* row_target,
                                void* R, bom_dtype r_dt, int64_t ldr,
                                float* loss, int32_t* n_valid, int32_t* flags, void* stream);

/* ------------------------------------------------------------------------------------------
 * bom_ema -- Sec. 3.2, Eq. (2) and Algorithm 1: q_t = beta1 q_{t-1} + (1 - beta1) s_t,
 * q_hat_t = q_t / (1 - beta1^t), with q_0 = 0 and t >= 1.
 *
 *   q      device fp32 [V], the state, updated in place.   s device fp32 [V].
 *   q_hat  device fp32 [V], output; must not overlap q.
 *   The factor 1/(1 - beta1^t) is formed on the host in fp64 and applied in fp32.
 * Errors: BOM_ERR_NULL, BOM_ERR_SHAPE (V < 1), BOM_ERR_HYPER (beta1 not in [0,1), t < 1),
 *         BOM_ERR_ALIAS, BOM_ERR_HIP.
 * ---------------------------------------------------------------------------------------- */
bom_status bom_ema(float* q, const float* s, int64_t V, float beta1, int64_t t, float* q_hat, void* stream);

/* ------------------------------------------------------------------------------------------
 * bom_head_vjp -- the output-head part of the single backward pass through the mixed
 * objective, Eq. (3), whose gradient is Eq. (4): u = (1 - lambda) g + lambda Jbar^T q_hat.
 * For the linear head z_i = W^T h_i (+ b), the gradient of L_mix with respect to the logits is
 *   G_ij = [i in I] ((1 - lambda) R_ij + lambda q_hat_j) / N_t        (q_hat held constant)
 * with R the residual rows of Sec. 3.2 (r_i = softmax(z_i) - onehot(y_i), Algorithm 1), and the head
 * products are
 *   dW = H^T G + dW_beta * dW     [d, V] (dW_beta = 0 overwrites; dW is not read then)
 *   db = (1 - lambda) s + lambda q_hat   [V]  (bias Jacobian = identity; equals 1^T G)
 *   dH = G W^T                     [N, d] of dh_dt
 * G is never written to memory. bf16 products use the equal rank-1 form
 *   dW = alpha H^T R + (sum_{i in I} H_i) (lambda q_hat / N_t)^T
 *   dH = alpha R W^T + 1_I (lambda / N_t W q_hat)^T
 * with alpha = (1 - lambda) / N_t, which multiplies R as stored and adds the history in fp32
 * (small products of both in one launch); small products with N or V above 8192 instead form G
 * tile by tile inside the GEMMs (the history folded into the output gradient at operand load,
 * rounded to bf16 for the MFMA), and fp32 inputs fold it in fp32.
 * N_t is read from the device word n_valid; when it is 0, G = 0.
 *
 * R_or_Z and is_residual: with is_residual = 1 the argument is R as bom_residual writes it (rows outside
 * I zero). With is_residual = 0 it is the logits Z, and the products form R themselves as their operand
 * copies pass through registers: R_ij = exp(z_ij - row_lse[i]) - [j == y_i] for rows in I, 0 for the
 * others, formed as bom_residual forms it for rows wider than one workgroup's registers (2^(z log2 e -
 * lse log2 e), minus 1 at the label) and rounded to dt once; it equals the stored R up to one rounding of
 * dt (bom_residual's narrow-row kernels scale exp(z - max) by 1/sum instead). bom_residual may then skip
 * writing R (R = NULL there): the step reads Z instead of writing and reading R, at the price of one
 * exponential per element of each operand copy.
 *
 *   H   device [N, ldh] of dt.   W device [d, ldw] of dt (the head as d x V).
 *   R_or_Z device [N, ldr] of dt.
 *   dt  BOM_BF16 (MFMA path, fp32 accumulation) or BOM_F32.
 *   labels device int32 [N] (defines I with ignore_index, as in bom_residual).
 *   row_lse device fp32 [N] (bom_residual's row_lse): read only when is_residual = 0, else may be NULL.
 *   q_hat device fp32 [V].   s device fp32 [V] (only read when db != NULL).
 *   n_valid device int32 [1].
 *   dW  device [d, lddw] of dw_dt; lddw >= V.   db device [V] of dw_dt, or NULL.
 *   dw_dt BOM_F32, or BOM_BF16 for bf16 gradient storage (dW, db formed in fp32 in the workspace, then
 *       rounded to nearest-even bf16: dW = bf16(H^T G + dW_beta * dW)).
 *   dH  device [N, lddh] of dh_dt (BOM_BF16 or BOM_F32), or NULL.
 *   workspace: at least bom_head_vjp_workspace_bytes(N, d, V, dt, dw_dt) bytes (may be 0).
 * Errors: BOM_ERR_NULL (also: row_lse missing with is_residual = 0), BOM_ERR_SHAPE (also: is_residual
 *         not 0 or 1), BOM_ERR_DTYPE, BOM_ERR_HYPER (lambda not in [0,1]), BOM_ERR_WORKSPACE, BOM_ERR_HIP.
 * ---------------------------------------------------------------------------------------- */
size_t bom_head_vjp_workspace_bytes(int64_t N, int64_t d, int64_t V, bom_dtype dt, bom_dtype dw_dt);
bom_status bom_head_vjp(const void* H, int64_t ldh, const void* W, int64_t ldw,
                        const void* R_or_Z, int32_t is_residual, int64_t ldr,
                        bom_dtype dt, int64_t N, int64_t d, int64_t V,
                        const int32_t* labels, int32_t ignore_index, const float* row_lse,
                        const float* q_hat, const float* s, const int32_t* n_valid, float lambda,
                        void* dW, bom_dtype dw_dt, int64_t lddw, float dW_beta,
                        void* db, void* dH, bom_dtype dh_dt, int64_t lddh,
                        void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------------------------
 * bom_update -- Sec. 3.4 and Algorithm 1 (the second-moment and parameter updates), over one flat fp32 buffer:
 *   u' = u_scale * u                       (or, when h != NULL: u_scale * ((1-lambda) u + lambda h))
 *   v  = beta2 v + (1 - beta2) u'^2,  v_hat = v / (1 - beta2^t)
 *   theta = (1 - lr * omega) theta - lr * u' / (sqrt(v_hat) + eps)
 * omega is the weight decay of the segment covering the element (the first match in `segs`),
 * else `weight_decay`. There is no first-moment buffer.
 *
 * BOM_V_FACTORED (a reading: the paper does not define it; Adafactor's rank-1 factorisation of
 * the same v): the buffer is viewed as a row-major matrix of block_cols columns (the last row may
 * be short) whose rows form blocks of block_rows rows. Per block:
 *   rho_i = sum_j u'_ij^2, kappa_j = sum_i u'_ij^2, Rr_i = beta2 Rr_i + (1-beta2) rho_i,
 *   Cc_j = beta2 Cc_j + (1-beta2) kappa_j, v_hat_ij = Rr_i Cc_j / sum_{k in block} Rr_k / (1-beta2^t)
 *   (0 when that sum is 0), then the same theta update.
 *
 *   theta device [P], in place.   u device [P].   h device [P] or NULL.   Their element type is
 *         fp32, or bf16 when cfg->state_dt = BOM_BF16 (dense layout only).
 *   v     dense: device [P] (in place), fp32 or bf16 like theta. factored: Rr, device fp32
 *         [ceil(P/block_cols)].
 *   v_col dense: NULL. factored: Cc, device fp32 [nblocks * block_cols],
 *         nblocks = ceil(ceil(P/block_cols) / block_rows).
 *   segs  HOST array of nsegs (<= BOM_MAX_SEGMENTS) segments inside [0, P), or NULL with nsegs 0.
 *   cfg   HOST struct. The factor 1/(1 - beta2^t) is formed on the host in fp64.
 *   workspace: at least bom_update_workspace_bytes(P, cfg) bytes (0 for the dense layout without
 *         clipping), 256-byte aligned.
 *
 * BOM_V_BLOCKS (Adam-mini's update map driven by the BOM numerator: Sec. 3.5 substitutes the numerator
 * into a base optimizer's map, and Adam-mini shares one second-moment value per block of parameters):
 * the segments must tile [0, P) in order (offset 0, each next offset the previous end, the last end P;
 * at most BOM_MAX_SEGMENTS per call, so a longer partition takes one call per run of segments on the
 * matching sub-ranges), and cfg->seg_blocks[k] >= 1 cuts segment k into consecutive blocks of that many
 * elements (the last one may be shorter). For block b with elements E_b:
 *   v_b = beta2 v_b + (1 - beta2) mean_{e in E_b} u'_e^2,  v_hat_b = v_b / (1 - beta2^t),
 *   theta_e = (1 - lr * omega) theta_e - lr * u'_e / (sqrt(v_hat_b) + eps).
 * Adam-mini's partition maps onto segments: one block per attention head (head_dim rows of a row-major
 * [out, in] weight), per output neuron (one row), per tensor (one block), or per element (block 1).
 *   v     device fp32 [sum_k ceil(length_k / seg_blocks[k])]: the blocks of segment 0, then 1, ...
 *   v_col NULL.  fp32 state only.
 *   workspace: at least bom_update_workspace_bytes(P, cfg) bytes (partial sums of blocks longer than
 *         4096 elements, bounded by P / 1024 + 64 floats, and the clipping pass).
 *
 * Global-norm clipping (cfg->clip_norm > 0; appendix "Pretraining Parameters" and appendix "Memory
 * and Timing Protocols" clip at 1.0, and appendix "Conditional Descent and Stationarity" counts the
 * clipping as part of the numerator supplied to the adaptive update): u' above is replaced by c u' with
 *   c = min(1, clip_norm / (||u'|| + 1e-6)),  ||u'|| the L2 norm of u' over all P elements,
 * computed on the device (no host synchronisation) and used by both the second moment and the step.
 * The 1e-6 guard is PyTorch's clip_grad_norm_ (the paper gives only the threshold). Dense layout:
 * one extra read of u (and h). Factored layout: no extra pass over u (the row statistics give the
 * norm). cfg->clip_stats, if not NULL, is a device fp32 [2] that receives ||u'|| and c.
 *
 * bf16 state storage (cfg->state_dt = BOM_BF16; appendix "NLP Fine-Tuning Parameters": bf16 parameter
 * and optimizer-state storage, the task-space EMA kept in fp32): theta, v, u and h are bf16; the step
 * is computed in fp32 from their values and theta and v are rounded to the nearest bf16 (ties to
 * even) when stored: 10 bytes per parameter instead of 20. Dense layout only (other layouts: BOM_ERR_DTYPE).
 * Errors: BOM_ERR_NULL, BOM_ERR_SHAPE, BOM_ERR_DTYPE, BOM_ERR_HYPER (beta2 not in [0,1), t < 1,
 *         eps <= 0, lambda not in [0,1], non-finite lr / u_scale / decay, clip_norm negative or not
 *         finite), BOM_ERR_ALIAS, BOM_ERR_WORKSPACE, BOM_ERR_HIP.
 * ---------------------------------------------------------------------------------------- */
typedef struct {
    int64_t offset;
    int64_t length;
    float weight_decay;
} bom_segment;

typedef struct {
    float lr, beta2, eps, lambda, u_scale;
    int64_t t;
    int32_t v_layout; /* BOM_V_DENSE, BOM_V_FACTORED or BOM_V_BLOCKS */
    int64_t block_rows, block_cols;
    float clip_norm;   /* > 0: global-norm clipping of the numerator at this norm; 0: none */
    float* clip_stats; /* device fp32 [2] or NULL: receives ||u'|| before clipping and the factor c */
    int32_t state_dt;  /* BOM_F32, or BOM_BF16: theta, v, u and h stored as bf16 (dense layout) */
    const int64_t* seg_blocks; /* BOM_V_BLOCKS: HOST array of nsegs block lengths; otherwise ignored */
} bom_update_cfg;

size_t bom_update_workspace_bytes(int64_t P, const bom_update_cfg* cfg);
bom_status bom_update(void* theta, void* v, float* v_col, const void* u, const void* h, int64_t P,
                      const bom_segment* segs, int32_t nsegs, float weight_decay, const bom_update_cfg* cfg,
                      void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------------------------
 * bom_adamw_update -- the comparison optimizer, not part of BOM's step: AdamW's update with its dense
 * first moment (Sec. 1: the EMA m of the gradients that BOM deletes; Sec. 3.5: the update map
 * a / (sqrt(v_hat) + eps) applied to m_hat = m / (1 - beta1^t)). It is the other arm of the first-order
 * cost model of appendix "First-order cost accounting" (Delta t = alpha N_out - beta P), timed beside
 * bom_update on the same buffers. With g' = u_scale * g:
 *   m = beta1 m + (1 - beta1) g';  v = beta2 v + (1 - beta2) g'^2 (dense), or the factored Rr, Cc of
 *   bom_update's BOM_V_FACTORED layout over g'^2;
 *   theta = (1 - lr * omega) theta - lr * (m / (1 - beta1^t)) / (sqrt(v_hat) + eps).
 * 28 bytes per parameter dense (read theta, m, v, g; write theta, m, v).
 *
 *   theta, m, g device fp32 [P] (theta, m in place).   v dense: device fp32 [P]; factored: Rr as in
 *   bom_update, with v_col = Cc.   segs, nsegs, weight_decay as in bom_update.   beta1 in [0, 1).
 *   cfg: lr, beta2, eps, u_scale, t, v_layout (BOM_V_DENSE, or BOM_V_FACTORED with block_cols 1024, 2048 or
 *   4096), block_rows, block_cols; clip_norm must be 0 and state_dt BOM_F32; lambda is not used.
 *   workspace: at least bom_update_workspace_bytes(P, cfg) bytes (0 for the dense layout).
 * Errors: BOM_ERR_NULL, BOM_ERR_SHAPE, BOM_ERR_HYPER, BOM_ERR_ALIAS, BOM_ERR_WORKSPACE, BOM_ERR_UNSUPPORTED,
 *         BOM_ERR_HIP.
 * ---------------------------------------------------------------------------------------- */
bom_status bom_adamw_update(float* theta, float* m, float* v, float* v_col, const float* g, int64_t P,
                            const bom_segment* segs, int32_t nsegs, float weight_decay, float beta1,
                            const bom_update_cfg* cfg, void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------------------------
 * bom_head_telemetry -- diagnostic beside the four steps (for telemetry steps only): the
 * historical-projection drift of the linear head, Sec. 3.3 Eq. (8) and appendix "Measuring historical
 * projection drift". For z_i = W^T h_i + b the batch-mean Jacobian maps a task-space x to
 * (hbar x^T, x), hbar = (1/N_t) sum_{i in I} H_i. One call, after bom_ema of the same step:
 *   M_W = beta1 M_W + (1 - beta1) hbar s^T,  M_b = beta1 M_b + (1 - beta1) s   (own-step projections)
 *   Mhat = M / (1 - beta1^t),  h = (hbar q_hat^T, q_hat)                     (BOM's reprojection)
 *   out[0] = cos(Mhat, h)   out[1] = ||Mhat - h|| / ||Mhat||   out[2] = ||s|| / ((1/N_t) sum_{i in I} ||r_i||)
 *   out[3] = ||Mhat||       out[4] = ||h||
 * The head is W and, when M_b is not NULL, b. Ratios with a zero denominator are reported as 0.
 *
 *   H  device [N, ldh] of h_dt.   R device [N, ldr] of r_dt (bom_residual's rows; rows outside I zero).
 *   labels, s, q_hat, n_valid as in bom_head_vjp.
 *   M_W device fp32 [d, ldm] (in place, zero before the first telemetry step); M_b device fp32 [V] or NULL.
 *   beta1 in [0, 1), t >= 1 the step counter of q (1/(1 - beta1^t) formed on the host in fp64).
 *   out device fp32 [5].   workspace: at least bom_head_telemetry_workspace_bytes(N, d, V) bytes.
 * Errors: BOM_ERR_NULL, BOM_ERR_SHAPE, BOM_ERR_DTYPE, BOM_ERR_HYPER, BOM_ERR_WORKSPACE, BOM_ERR_ALIAS,
 *         BOM_ERR_HIP.
 * ---------------------------------------------------------------------------------------- */
size_t bom_head_telemetry_workspace_bytes(int64_t N, int64_t d, int64_t V);
bom_status bom_head_telemetry(const void* H, int64_t ldh, bom_dtype h_dt, const void* R, int64_t ldr, bom_dtype r_dt,
                              int64_t N, int64_t d, int64_t V, const int32_t* labels, int32_t ignore_index,
                              const float* s, const float* q_hat, const int32_t* n_valid, float* M_W, int64_t ldm,
                              float* M_b, float beta1, int64_t t, float* out, void* workspace, size_t ws_bytes,
                              void* stream);

/* ------------------------------------------------------------------------------------------
 * bom_head_forward -- support call (row a0 of the path; the forward is common work, not one of the
 * four steps): the linear head's logits Z = H W (+ b), fp32 accumulation, Z rounded once to dt.
 * dt = BOM_BF16 (the language-model and vision workloads' logits, as bf16 autocast computes them) runs
 * on the matrix cores (256 x 256 tiles) when d and V are multiples of 8 and H, W are 16-byte aligned
 * with leading dimensions that are multiples of 8, and on a SIMT kernel otherwise; dt = BOM_F32
 * (the tiny classifier) runs on the SIMT kernel.
 *   H device [N, ldh], W device [d, ldw], b device [V] or NULL, Z device [N, ldz], all of dt.
 * Errors: BOM_ERR_NULL, BOM_ERR_SHAPE, BOM_ERR_DTYPE, BOM_ERR_HIP.
 * ---------------------------------------------------------------------------------------- */
bom_status bom_head_forward(const void* H, int64_t ldh, const void* W, int64_t ldw, const void* b, bom_dtype dt,
                            int64_t N, int64_t d, int64_t V, void* Z, int64_t ldz, void* stream);

/* ------------------------------------------------------------------------------------------
 * bom_head_forward_residual -- the head forward and bom_residual in one call (appendix "First-order cost
 * accounting": the output-side work over N_out = N V coordinates is where BOM's bookkeeping sits).
 * Computes Z = H W (+ b) as bom_head_forward does and then every output of bom_residual on that Z.
 * For bf16 on the matrix cores (d and V multiples of 8, 16-byte aligned H, W, Z and R with leading
 * dimensions that are multiples of 8) the forward's epilogue also reduces each 256-column tile of every
 * row of the rounded logits (maximum, first column reaching it, sum of exp(z - max)) and records the
 * target logit, so the residual only merges those records per row and re-reads Z once for R and the
 * column sums: no row is split across workgroups and no row statistics pass is made over Z. Other shapes
 * and fp32 run the forward, then bom_residual.
 *
 *   H, ldh, W, ldw, b, dt, N, d, V, Z, ldz: as bom_head_forward (Z is written).
 *   labels, ignore_index, s, row_lse, row_argmax (nullable), row_target (required here), R (nullable), ldr,
 *   loss, n_valid, flags: as bom_residual (r_dt = dt).
 *   workspace: at least bom_head_forward_residual_workspace_bytes(N, V, dt) bytes, 256-byte aligned.
 * Errors: BOM_ERR_NULL, BOM_ERR_SHAPE, BOM_ERR_DTYPE, BOM_ERR_WORKSPACE, BOM_ERR_ALIAS, BOM_ERR_HIP.
 * ---------------------------------------------------------------------------------------- */
size_t bom_head_forward_residual_workspace_bytes(int64_t N, int64_t V, bom_dtype dt);
bom_status bom_head_forward_residual(const void* H, int64_t ldh, const void* W, int64_t ldw, const void* b,
                                     bom_dtype dt, int64_t N, int64_t d, int64_t V, void* Z, int64_t ldz,
                                     const int32_t* labels, int32_t ignore_index,
                                     float* s, float* row_lse, int32_t* row_argmax, float* row_target,
                                     void* R, int64_t ldr, float* loss, int32_t* n_valid, int32_t* flags,
                                     void* workspace, size_t ws_bytes, void* stream);

/* Environment variables, each read once per process on first use (for measurement and tests; results do
 * not depend on them beyond rounding order):
 *   BOM_VJP_WAVES = "dH,dW,fwd,pair"  waves per workgroup (4 or 8) of the 256-tile products; default 8,8,8,8.
 *   BOM_VJP_PLAN  = "kw,sw,kh,sh"     force a head-VJP kernel kind and k split per product (A/B runs only).
 *   BOM_VJP_XCD_BLOCK = 0             the plain XCD tile order of the 256-tile products instead of the
 *                                      blocked one (4 outer x 8 inner tiles per XCD round; the same sums).
 *   BOM_RESIDUAL_SPIN = n             poll bound of the split-row residual exchange; negative: every part
 *                                      recomputes its partners' row records from Z (the fallback path).
 */

/* Static text of a status code, and the thread-local detail of the last failure ("" if none). */
const char* bom_status_string(bom_status status);
const char* bom_last_error(void);
/* Library ABI version (major * 10000 + minor * 100 + patch). */
int32_t bom_version(void);
/* Identity of the sources the library was built from: the first 16 hex digits of a SHA-256 over the
 * names and contents of the HIP sources, their headers and this header (static text). */
const char* bom_build_id(void);

#ifdef __cplusplus
}
#endif
#endif /* BOM_H */
