// C-ABI of libbom.so (declared in include/bom.h): host-side validation, then enqueue.
// Every argument error is returned before any HIP call; no exception crosses the ABI.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "bom.h"
#include "kernels.hpp"

namespace {

thread_local char g_last_error[512] = "";

bom_status fail(bom_status st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return st;
}

bom_status hip_status(hipError_t e, const char* where) {
    if (e == hipSuccess) {
        g_last_error[0] = '\0';
        return BOM_OK;
    }
    return fail(BOM_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

constexpr int64_t kMaxDim = (int64_t)1 << 31;

bool is_dtype(bom_dtype d) { return d == BOM_F32 || d == BOM_BF16; }

bool overlap(const void* a, size_t na, const void* b, size_t nb) {
    const char* pa = static_cast<const char*>(a);
    const char* pb = static_cast<const char*>(b);
    return pa < pb + nb && pb < pa + na;
}

bool finite(float x) { return std::isfinite(x); }

}  // namespace

extern "C" {

const char* bom_status_string(bom_status s) {
    switch (s) {
        case BOM_OK: return "BOM_OK";
        case BOM_ERR_NULL: return "BOM_ERR_NULL: a required pointer is NULL";
        case BOM_ERR_SHAPE: return "BOM_ERR_SHAPE: a size or leading dimension is out of range";
        case BOM_ERR_DTYPE: return "BOM_ERR_DTYPE: unsupported dtype combination";
        case BOM_ERR_HYPER: return "BOM_ERR_HYPER: a hyperparameter is outside its domain";
        case BOM_ERR_WORKSPACE: return "BOM_ERR_WORKSPACE: workspace missing or too small";
        case BOM_ERR_ALIAS: return "BOM_ERR_ALIAS: buffers that must be distinct overlap";
        case BOM_ERR_HIP: return "BOM_ERR_HIP: a HIP runtime call failed";
        case BOM_ERR_UNSUPPORTED: return "BOM_ERR_UNSUPPORTED: not implemented by this library";
    }
    return "unknown bom_status";
}

const char* bom_last_error(void) { return g_last_error; }

int32_t bom_version(void) { return 30000; }

#ifndef BOM_BUILD_ID
#define BOM_BUILD_ID "unknown"
#endif
const char* bom_build_id(void) { return BOM_BUILD_ID; }

size_t bom_residual_workspace_bytes(int64_t N, int64_t V, bom_dtype z_dt) {
    if (N < 1 || V < 1 || N >= kMaxDim || V >= kMaxDim || !is_dtype(z_dt)) return 0;
    return bom::residual_workspace_bytes(N, V, z_dt);
}

}  // extern "C"

namespace {
// Argument checks of bom_residual (also run by the allocation-free variant before it touches the device).
bom_status bom_residual_validate(const void* Z, bom_dtype z_dt, int64_t N, int64_t V, int64_t ldz,
                                 const int32_t* labels, const float* s, const float* row_lse, const void* R,
                                 bom_dtype r_dt, int64_t ldr, const float* loss, const int32_t* n_valid,
                                 const int32_t* flags, const void* workspace, size_t ws_bytes) {
    if (!Z || !labels || !s || !row_lse || !loss || !n_valid || !flags)
        return fail(BOM_ERR_NULL, "bom_residual: Z, labels, s, row_lse, loss, n_valid and flags are required");
    if (N < 1 || V < 2 || N >= kMaxDim || V >= kMaxDim)
        return fail(BOM_ERR_SHAPE, "bom_residual: need 1 <= N < 2^31 and 2 <= V < 2^31 (N=%lld V=%lld)", (long long)N,
                    (long long)V);
    if (ldz < V || (R && ldr < V))
        return fail(BOM_ERR_SHAPE, "bom_residual: leading dimensions must be >= V (ldz=%lld ldr=%lld V=%lld)",
                    (long long)ldz, (long long)ldr, (long long)V);
    if (!is_dtype(z_dt) || (R && r_dt != z_dt))
        return fail(BOM_ERR_DTYPE, "bom_residual: z_dt must be BOM_F32 or BOM_BF16 and r_dt must equal it");
    const size_t need = bom::residual_workspace_bytes(N, V, z_dt);
    if (!workspace || ws_bytes < need)
        return fail(BOM_ERR_WORKSPACE, "bom_residual: workspace needs %zu bytes, got %zu", need, ws_bytes);
    if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
        return fail(BOM_ERR_WORKSPACE, "bom_residual: workspace must be 256-byte aligned");
    const size_t esz = z_dt == BOM_BF16 ? 2 : 4;
    if (R && overlap(R, (size_t)((N - 1) * ldr + V) * esz, Z, (size_t)((N - 1) * ldz + V) * esz))
        return fail(BOM_ERR_ALIAS, "bom_residual: R must not overlap Z");
    return BOM_OK;
}
}  // namespace

extern "C" {

bom_status bom_residual(const void* Z, bom_dtype z_dt, int64_t N, int64_t V, int64_t ldz, const int32_t* labels,
                        int32_t ignore_index, float* s, float* row_lse, int32_t* row_argmax, float* row_target, void* R,
                        bom_dtype r_dt, int64_t ldr, float* loss, int32_t* n_valid, int32_t* flags, void* workspace,
                        size_t ws_bytes, void* stream) {
    const bom_status st = bom_residual_validate(Z, z_dt, N, V, ldz, labels, s, row_lse, R, r_dt, ldr, loss, n_valid,
                                                flags, workspace, ws_bytes);
    if (st != BOM_OK) return st;
    hipError_t e = bom::launch_residual(Z, z_dt, (int)N, (int)V, ldz, labels, ignore_index, s, row_lse, row_argmax,
                                        row_target, R, ldr, loss, n_valid, flags, workspace,
                                        static_cast<hipStream_t>(stream));
    return hip_status(e, "bom_residual");
}

bom_status bom_residual_noalloc(const void* Z, bom_dtype z_dt, int64_t N, int64_t V, int64_t ldz,
                                const int32_t* labels, int32_t ignore_index, float* s, float* row_lse,
                                int32_t* row_argmax, float* row_target, void* R, bom_dtype r_dt, int64_t ldr,
                                float* loss, int32_t* n_valid, int32_t* flags, void* stream) {
    if (N >= 1 && V >= 2 && N < kMaxDim && V < kMaxDim && is_dtype(z_dt)) {
        const size_t need = bom::residual_workspace_bytes(N, V, z_dt);
        if (need > bom::kResidualScratchBytes)
            return fail(BOM_ERR_WORKSPACE,
                        "bom_residual_noalloc: this shape needs %zu bytes of scratch; the library's fixed scratch "
                        "holds %zu (use bom_residual with a workspace)",
                        need, bom::kResidualScratchBytes);
    }
    // the arguments are validated by bom_residual before anything touches the device: look the scratch
    // up only for a call that passes them
    const size_t big = bom::kResidualScratchBytes;
    void* probe = reinterpret_cast<void*>((uintptr_t)256);   // aligned stand-in, never dereferenced
    bom_status st = bom_residual_validate(Z, z_dt, N, V, ldz, labels, s, row_lse, R, r_dt, ldr, loss, n_valid, flags,
                                          probe, big);
    if (st != BOM_OK) return st;
    void* ws = nullptr;
    const hipError_t e = bom::residual_scratch(&ws);
    if (e != hipSuccess) return hip_status(e, "bom_residual_noalloc (scratch lookup)");
    return bom_residual(Z, z_dt, N, V, ldz, labels, ignore_index, s, row_lse, row_argmax, row_target, R, r_dt, ldr,
                        loss, n_valid, flags, ws, big, stream);
}

bom_status bom_ema(float* q, const float* s, int64_t V, float beta1, int64_t t, float* q_hat, void* stream) {
    if (!q || !s || !q_hat) return fail(BOM_ERR_NULL, "bom_ema: q, s and q_hat are required");
    if (V < 1 || V >= kMaxDim) return fail(BOM_ERR_SHAPE, "bom_ema: need 1 <= V < 2^31");
    if (!(beta1 >= 0.f && beta1 < 1.f) || t < 1)
        return fail(BOM_ERR_HYPER, "bom_ema: need beta1 in [0, 1) and t >= 1 (beta1=%g t=%lld)", (double)beta1,
                    (long long)t);
    if (overlap(q, (size_t)V * 4, q_hat, (size_t)V * 4)) return fail(BOM_ERR_ALIAS, "bom_ema: q_hat must not overlap q");
    const double bc = 1.0 - std::pow((double)beta1, (double)t);
    const float inv_bc1 = (float)(1.0 / bc);
    return hip_status(bom::launch_ema(q, s, V, beta1, inv_bc1, q_hat, static_cast<hipStream_t>(stream)), "bom_ema");
}

size_t bom_head_vjp_workspace_bytes(int64_t N, int64_t d, int64_t V, bom_dtype dt, bom_dtype dw_dt) {
    if (N < 1 || d < 1 || V < 1 || N >= kMaxDim || d >= kMaxDim || V >= kMaxDim || !is_dtype(dt) || !is_dtype(dw_dt))
        return 0;
    return bom::head_vjp_workspace_bytes(N, d, V, dt, dw_dt);
}

bom_status bom_head_vjp(const void* H, int64_t ldh, const void* W, int64_t ldw, const void* R, int32_t is_residual,
                        int64_t ldr, bom_dtype dt, int64_t N, int64_t d, int64_t V, const int32_t* labels,
                        int32_t ignore_index, const float* row_lse, const float* q_hat, const float* s,
                        const int32_t* n_valid, float lambda, void* dW, bom_dtype dw_dt, int64_t lddw, float dW_beta,
                        void* db, void* dH, bom_dtype dh_dt, int64_t lddh, void* workspace, size_t ws_bytes,
                        void* stream) {
    if (!H || !W || !R || !labels || !q_hat || !n_valid || !dW)
        return fail(BOM_ERR_NULL, "bom_head_vjp: H, W, R_or_Z, labels, q_hat, n_valid and dW are required");
    if (db && !s) return fail(BOM_ERR_NULL, "bom_head_vjp: s is required when db is requested");
    if (is_residual != 0 && is_residual != 1)
        return fail(BOM_ERR_SHAPE, "bom_head_vjp: is_residual must be 1 (R) or 0 (logits Z)");
    if (!is_residual && !row_lse) return fail(BOM_ERR_NULL, "bom_head_vjp: row_lse is required with the logits Z");
    if (N < 1 || d < 1 || V < 2 || N >= kMaxDim || d >= kMaxDim || V >= kMaxDim)
        return fail(BOM_ERR_SHAPE, "bom_head_vjp: need N >= 1, d >= 1, V >= 2, all < 2^31");
    if (ldh < d || ldw < V || ldr < V || lddw < V || (dH && lddh < d))
        return fail(BOM_ERR_SHAPE, "bom_head_vjp: a leading dimension is smaller than its row length");
    if ((int64_t)d * V >= ((int64_t)1 << 40) || (int64_t)N * d >= ((int64_t)1 << 40))
        return fail(BOM_ERR_SHAPE, "bom_head_vjp: output too large");
    if (!is_dtype(dt) || !is_dtype(dw_dt) || (dH && !is_dtype(dh_dt)))
        return fail(BOM_ERR_DTYPE, "bom_head_vjp: unsupported dtype");
    if (!(lambda >= 0.f && lambda <= 1.f)) return fail(BOM_ERR_HYPER, "bom_head_vjp: need lambda in [0, 1]");
    if (!finite(dW_beta)) return fail(BOM_ERR_HYPER, "bom_head_vjp: dW_beta must be finite");
    const size_t need = bom::head_vjp_workspace_bytes(N, d, V, dt, dw_dt);
    if (need > 0 && (!workspace || ws_bytes < need))
        return fail(BOM_ERR_WORKSPACE, "bom_head_vjp: workspace needs %zu bytes, got %zu", need, ws_bytes);
    if (workspace && reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
        return fail(BOM_ERR_WORKSPACE, "bom_head_vjp: workspace must be 256-byte aligned");
    bom::HeadVjpArgs a{H, ldh, W, ldw, R, ldr, is_residual, row_lse, dt, (int)N, (int)d, (int)V, labels, ignore_index,
                       q_hat, s, n_valid, lambda, dW, dw_dt, lddw, dW_beta, db, dH, dh_dt, lddh, workspace, ws_bytes};
    return hip_status(bom::launch_head_vjp(a, static_cast<hipStream_t>(stream)), "bom_head_vjp");
}

size_t bom_update_workspace_bytes(int64_t P, const bom_update_cfg* cfg) { return bom::update_workspace_bytes(P, cfg); }

bom_status bom_update(void* theta_p, void* v_p, float* v_col, const void* u_p, const void* h_p, int64_t P,
                      const bom_segment* segs, int32_t nsegs, float weight_decay, const bom_update_cfg* cfg,
                      void* workspace, size_t ws_bytes, void* stream) {
    if (!theta_p || !v_p || !u_p || !cfg) return fail(BOM_ERR_NULL, "bom_update: theta, v, u and cfg are required");
    if (P < 1) return fail(BOM_ERR_SHAPE, "bom_update: need P >= 1");
    if (nsegs < 0 || nsegs > BOM_MAX_SEGMENTS || (nsegs > 0 && !segs))
        return fail(BOM_ERR_SHAPE, "bom_update: need 0 <= nsegs <= %d and segs when nsegs > 0", BOM_MAX_SEGMENTS);
    const bom_update_cfg& c = *cfg;
    if (!(c.beta2 >= 0.f && c.beta2 < 1.f) || c.t < 1 || !(c.eps > 0.f) || !finite(c.eps) || !finite(c.lr) ||
        !(c.lambda >= 0.f && c.lambda <= 1.f) || !finite(c.u_scale) || !finite(weight_decay) ||
        !(c.clip_norm >= 0.f) || !finite(c.clip_norm))
        return fail(BOM_ERR_HYPER, "bom_update: need beta2 in [0,1), t >= 1, eps > 0, lambda in [0,1], finite lr, "
                                   "u_scale and weight decay, and a finite clip_norm >= 0");
    bom::SegTable st{};
    st.n = nsegs;
    st.wd_default = weight_decay;
    for (int k = 0; k < nsegs; ++k) {
        const bom_segment& g = segs[k];
        if (g.offset < 0 || g.length < 0 || g.offset + g.length > P)
            return fail(BOM_ERR_SHAPE, "bom_update: segment %d [%lld, +%lld) is outside [0, P)", k, (long long)g.offset,
                        (long long)g.length);
        if (!finite(g.weight_decay)) return fail(BOM_ERR_HYPER, "bom_update: segment %d decay is not finite", k);
        st.begin[k] = g.offset;
        st.end[k] = g.offset + g.length;
        st.wd[k] = g.weight_decay;
    }
    bom::UpdateScalars sc;
    sc.lr = c.lr;
    sc.beta2 = c.beta2;
    sc.one_minus_beta2 = (float)(1.0 - (double)c.beta2);
    sc.eps = c.eps;
    sc.lambda = c.lambda;
    sc.u_scale = c.u_scale;
    sc.inv_bc2 = (float)(1.0 / (1.0 - std::pow((double)c.beta2, (double)c.t)));
    sc.clip_norm = c.clip_norm;
    sc.clip = nullptr;   // set by the launcher once the clipping pass is enqueued
    sc.clip_stats = c.clip_norm > 0.f ? c.clip_stats : nullptr;
    if (c.state_dt != BOM_F32 && c.state_dt != BOM_BF16)
        return fail(BOM_ERR_DTYPE, "bom_update: state_dt must be BOM_F32 or BOM_BF16");
    if (c.state_dt == BOM_BF16 && c.v_layout != BOM_V_DENSE)
        return fail(BOM_ERR_DTYPE, "bom_update: bf16 state storage is implemented for the dense layout only");
    const size_t pb = (size_t)P * (c.state_dt == BOM_BF16 ? 2 : 4);
    if (overlap(theta_p, pb, u_p, pb) || (h_p && overlap(theta_p, pb, h_p, pb)))
        return fail(BOM_ERR_ALIAS, "bom_update: theta must not overlap u or h");
    hipStream_t strm = static_cast<hipStream_t>(stream);
    if (c.state_dt == BOM_BF16) {
        if (v_col) return fail(BOM_ERR_SHAPE, "bom_update: v_col must be NULL for the dense layout");
        if (overlap(v_p, pb, theta_p, pb) || overlap(v_p, pb, u_p, pb) || (h_p && overlap(v_p, pb, h_p, pb)))
            return fail(BOM_ERR_ALIAS, "bom_update: v must not overlap theta, u or h");
        const size_t need_b = bom::update_workspace_bytes(P, cfg);
        if (need_b > 0) {
            if (!workspace || ws_bytes < need_b)
                return fail(BOM_ERR_WORKSPACE, "bom_update: workspace needs %zu bytes, got %zu", need_b, ws_bytes);
            if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
                return fail(BOM_ERR_WORKSPACE, "bom_update: workspace must be 256-byte aligned");
        }
        return hip_status(bom::launch_update_dense_bf16(static_cast<uint16_t*>(theta_p), static_cast<uint16_t*>(v_p),
                                                        static_cast<const uint16_t*>(u_p),
                                                        static_cast<const uint16_t*>(h_p), P, st, sc, workspace, strm),
                          "bom_update");
    }
    float* theta = static_cast<float*>(theta_p);
    float* v = static_cast<float*>(v_p);
    const float* u = static_cast<const float*>(u_p);
    const float* h = static_cast<const float*>(h_p);
    if (c.v_layout == BOM_V_DENSE) {
        if (v_col) return fail(BOM_ERR_SHAPE, "bom_update: v_col must be NULL for the dense layout");
        if (overlap(v, pb, theta, pb) || overlap(v, pb, u, pb) || (h && overlap(v, pb, h, pb)))
            return fail(BOM_ERR_ALIAS, "bom_update: v must not overlap theta, u or h");
        const size_t need_d = bom::update_workspace_bytes(P, cfg);
        if (need_d > 0) {
            if (!workspace || ws_bytes < need_d)
                return fail(BOM_ERR_WORKSPACE, "bom_update: workspace needs %zu bytes, got %zu", need_d, ws_bytes);
            if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
                return fail(BOM_ERR_WORKSPACE, "bom_update: workspace must be 256-byte aligned");
        }
        return hip_status(bom::launch_update_dense(theta, v, u, h, P, st, sc, workspace, strm), "bom_update");
    }
    if (c.v_layout == BOM_V_BLOCKS) {
        if (v_col) return fail(BOM_ERR_SHAPE, "bom_update: v_col must be NULL for the block layout");
        if (nsegs < 1 || !c.seg_blocks)
            return fail(BOM_ERR_NULL, "bom_update: the block layout needs segments and cfg->seg_blocks");
        bom::BlockSegs bs{};
        bs.n = nsegs;
        int64_t pos = 0;
        for (int k = 0; k < nsegs; ++k) {
            if (segs[k].offset != pos || segs[k].length < 1)
                return fail(BOM_ERR_SHAPE, "bom_update: block layout segments must tile [0, P) in order (segment %d)", k);
            if (c.seg_blocks[k] < 1) return fail(BOM_ERR_SHAPE, "bom_update: segment %d block length must be >= 1", k);
            bs.begin[k] = pos;
            bs.len[k] = segs[k].length;
            bs.blk[k] = c.seg_blocks[k];
            bs.wd[k] = segs[k].weight_decay;
            pos += segs[k].length;
        }
        if (pos != P) return fail(BOM_ERR_SHAPE, "bom_update: block layout segments end at %lld, not P", (long long)pos);
        const size_t vb = (size_t)bom::blocks_count(bs) * 4;
        if (overlap(v, vb, theta, pb) || overlap(v, vb, u, pb) || (h && overlap(v, vb, h, pb)))
            return fail(BOM_ERR_ALIAS, "bom_update: v must not overlap theta, u or h");
        const size_t need_k = bom::update_workspace_bytes(P, cfg);
        if (!workspace || ws_bytes < need_k)
            return fail(BOM_ERR_WORKSPACE, "bom_update: workspace needs %zu bytes, got %zu", need_k, ws_bytes);
        if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
            return fail(BOM_ERR_WORKSPACE, "bom_update: workspace must be 256-byte aligned");
        return hip_status(bom::launch_update_blocks(theta, v, u, h, P, bs, sc, workspace, strm), "bom_update");
    }
    if (c.v_layout != BOM_V_FACTORED) return fail(BOM_ERR_SHAPE, "bom_update: unknown v_layout %d", c.v_layout);
    if (!v_col) return fail(BOM_ERR_NULL, "bom_update: the factored layout needs v_col");
    if (c.block_rows < 1 || c.block_cols < 4 || c.block_cols > 16384 || c.block_cols % 4 != 0)
        return fail(BOM_ERR_UNSUPPORTED, "bom_update: factored layout needs block_rows >= 1 and block_cols a multiple "
                                         "of 4 in [4, 16384]");
    if (P % 4 != 0) return fail(BOM_ERR_UNSUPPORTED, "bom_update: factored layout needs P % 4 == 0");
    auto al = [](const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; };
    if (!al(theta) || !al(u) || (h && !al(h)) || !al(v_col))
        return fail(BOM_ERR_UNSUPPORTED, "bom_update: factored layout needs 16-byte aligned theta, u, h and v_col");
    const size_t need = bom::update_workspace_bytes(P, cfg);
    if (!workspace || ws_bytes < need)
        return fail(BOM_ERR_WORKSPACE, "bom_update: workspace needs %zu bytes, got %zu", need, ws_bytes);
    if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
        return fail(BOM_ERR_WORKSPACE, "bom_update: workspace must be 256-byte aligned");
    const int64_t nrows = (P + c.block_cols - 1) / c.block_cols;
    const int64_t nblocks = (nrows + c.block_rows - 1) / c.block_rows;
    if (overlap(v, (size_t)nrows * 4, v_col, (size_t)nblocks * c.block_cols * 4) || overlap(v, (size_t)nrows * 4, theta, pb) ||
        overlap(v_col, (size_t)nblocks * c.block_cols * 4, theta, pb))
        return fail(BOM_ERR_ALIAS, "bom_update: Rr, Cc and theta must be distinct");
    return hip_status(bom::launch_update_factored(theta, v, v_col, u, h, P, c.block_rows, c.block_cols, st, sc, workspace,
                                                  strm),
                      "bom_update");
}

bom_status bom_adamw_update(float* theta, float* m, float* v, float* v_col, const float* g, int64_t P,
                            const bom_segment* segs, int32_t nsegs, float weight_decay, float beta1,
                            const bom_update_cfg* cfg, void* workspace, size_t ws_bytes, void* stream) {
    if (!theta || !m || !v || !g || !cfg) return fail(BOM_ERR_NULL, "bom_adamw_update: theta, m, v, g and cfg are required");
    if (P < 1) return fail(BOM_ERR_SHAPE, "bom_adamw_update: need P >= 1");
    if (nsegs < 0 || nsegs > BOM_MAX_SEGMENTS || (nsegs > 0 && !segs))
        return fail(BOM_ERR_SHAPE, "bom_adamw_update: need 0 <= nsegs <= %d and segs when nsegs > 0", BOM_MAX_SEGMENTS);
    const bom_update_cfg& c = *cfg;
    if (!(beta1 >= 0.f && beta1 < 1.f) || !(c.beta2 >= 0.f && c.beta2 < 1.f) || c.t < 1 || !(c.eps > 0.f) ||
        !finite(c.eps) || !finite(c.lr) || !finite(c.u_scale) || !finite(weight_decay))
        return fail(BOM_ERR_HYPER, "bom_adamw_update: need beta1, beta2 in [0,1), t >= 1, eps > 0, finite lr, u_scale "
                                   "and weight decay");
    if (c.clip_norm != 0.f || c.state_dt != BOM_F32 || (c.v_layout != BOM_V_DENSE && c.v_layout != BOM_V_FACTORED))
        return fail(BOM_ERR_UNSUPPORTED, "bom_adamw_update: fp32 state, the dense or factored layout, no clipping");
    bom::SegTable st{};
    st.n = nsegs;
    st.wd_default = weight_decay;
    for (int k = 0; k < nsegs; ++k) {
        const bom_segment& sg = segs[k];
        if (sg.offset < 0 || sg.length < 0 || sg.offset + sg.length > P)
            return fail(BOM_ERR_SHAPE, "bom_adamw_update: segment %d is outside [0, P)", k);
        if (!finite(sg.weight_decay)) return fail(BOM_ERR_HYPER, "bom_adamw_update: segment %d decay is not finite", k);
        st.begin[k] = sg.offset;
        st.end[k] = sg.offset + sg.length;
        st.wd[k] = sg.weight_decay;
    }
    bom::UpdateScalars sc{};
    sc.lr = c.lr;
    sc.beta2 = c.beta2;
    sc.one_minus_beta2 = (float)(1.0 - (double)c.beta2);
    sc.eps = c.eps;
    sc.lambda = 0.f;
    sc.u_scale = c.u_scale;
    sc.inv_bc2 = (float)(1.0 / (1.0 - std::pow((double)c.beta2, (double)c.t)));
    sc.clip_norm = 0.f;
    sc.clip = nullptr;
    sc.clip_stats = nullptr;
    sc.beta1 = beta1;
    sc.one_minus_beta1 = (float)(1.0 - (double)beta1);
    sc.inv_bc1 = (float)(1.0 / (1.0 - std::pow((double)beta1, (double)c.t)));
    const size_t pb = (size_t)P * 4;
    if (overlap(theta, pb, g, pb) || overlap(m, pb, theta, pb) || overlap(m, pb, g, pb))
        return fail(BOM_ERR_ALIAS, "bom_adamw_update: theta, m and g must be distinct");
    hipStream_t strm = static_cast<hipStream_t>(stream);
    if (c.v_layout == BOM_V_DENSE) {
        if (v_col) return fail(BOM_ERR_SHAPE, "bom_adamw_update: v_col must be NULL for the dense layout");
        if (overlap(v, pb, theta, pb) || overlap(v, pb, m, pb) || overlap(v, pb, g, pb))
            return fail(BOM_ERR_ALIAS, "bom_adamw_update: v must not overlap theta, m or g");
        return hip_status(bom::launch_adamw_dense(theta, m, v, g, P, st, sc, strm), "bom_adamw_update");
    }
    if (!v_col) return fail(BOM_ERR_NULL, "bom_adamw_update: the factored layout needs v_col");
    if (c.block_rows < 1 || (c.block_cols != 1024 && c.block_cols != 2048 && c.block_cols != 4096))
        return fail(BOM_ERR_UNSUPPORTED, "bom_adamw_update: factored layout needs block_cols of 1024, 2048 or 4096");
    auto al = [](const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; };
    if (P % 4 != 0 || !al(theta) || !al(m) || !al(g) || !al(v_col))
        return fail(BOM_ERR_UNSUPPORTED, "bom_adamw_update: factored layout needs P % 4 == 0 and 16-byte aligned arrays");
    const size_t need = bom::update_workspace_bytes(P, cfg);
    if (!workspace || ws_bytes < need)
        return fail(BOM_ERR_WORKSPACE, "bom_adamw_update: workspace needs %zu bytes, got %zu", need, ws_bytes);
    if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
        return fail(BOM_ERR_WORKSPACE, "bom_adamw_update: workspace must be 256-byte aligned");
    const int64_t nrows = (P + c.block_cols - 1) / c.block_cols;
    const int64_t nblocks = (nrows + c.block_rows - 1) / c.block_rows;
    if (overlap(v, (size_t)nrows * 4, v_col, (size_t)nblocks * c.block_cols * 4) || overlap(v, (size_t)nrows * 4, theta, pb) ||
        overlap(v_col, (size_t)nblocks * c.block_cols * 4, theta, pb))
        return fail(BOM_ERR_ALIAS, "bom_adamw_update: Rr, Cc and theta must be distinct");
    return hip_status(bom::launch_adamw_factored(theta, m, v, v_col, g, P, c.block_rows, c.block_cols, st, sc, workspace,
                                                 strm),
                      "bom_adamw_update");
}

size_t bom_head_forward_residual_workspace_bytes(int64_t N, int64_t V, bom_dtype dt) {
    if (N < 1 || V < 2 || N >= kMaxDim || V >= kMaxDim || !is_dtype(dt)) return 0;
    const size_t a = bom::residual_from_stats_workspace_bytes(N, V), b = bom::residual_workspace_bytes(N, V, dt);
    return a > b ? a : b;
}

bom_status bom_head_forward_residual(const void* H, int64_t ldh, const void* W, int64_t ldw, const void* b, bom_dtype dt,
                                     int64_t N, int64_t d, int64_t V, void* Z, int64_t ldz, const int32_t* labels,
                                     int32_t ignore_index, float* s, float* row_lse, int32_t* row_argmax,
                                     float* row_target, void* R, int64_t ldr, float* loss, int32_t* n_valid,
                                     int32_t* flags, void* workspace, size_t ws_bytes, void* stream) {
    if (!H || !W || !Z || !labels || !s || !row_lse || !row_target || !loss || !n_valid || !flags)
        return fail(BOM_ERR_NULL, "bom_head_forward_residual: H, W, Z, labels, s, row_lse, row_target, loss, n_valid "
                                  "and flags are required");
    if (N < 1 || d < 1 || V < 2 || N >= kMaxDim || d >= kMaxDim || V >= kMaxDim)
        return fail(BOM_ERR_SHAPE, "bom_head_forward_residual: need N >= 1, d >= 1, V >= 2, all < 2^31");
    if (ldh < d || ldw < V || ldz < V || (R && ldr < V))
        return fail(BOM_ERR_SHAPE, "bom_head_forward_residual: a leading dimension is smaller than its row length");
    if (!is_dtype(dt)) return fail(BOM_ERR_DTYPE, "bom_head_forward_residual: dt must be BOM_F32 or BOM_BF16");
    const size_t need = bom_head_forward_residual_workspace_bytes(N, V, dt);
    if (!workspace || ws_bytes < need)
        return fail(BOM_ERR_WORKSPACE, "bom_head_forward_residual: workspace needs %zu bytes, got %zu", need, ws_bytes);
    if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
        return fail(BOM_ERR_WORKSPACE, "bom_head_forward_residual: workspace must be 256-byte aligned");
    const size_t esz = dt == BOM_BF16 ? 2 : 4;
    const size_t zb = (size_t)((N - 1) * ldz + V) * esz;
    if ((R && overlap(R, (size_t)((N - 1) * ldr + V) * esz, Z, zb)) || overlap(Z, zb, H, (size_t)((N - 1) * ldh + d) * esz) ||
        overlap(Z, zb, W, (size_t)((d - 1) * ldw + V) * esz))
        return fail(BOM_ERR_ALIAS, "bom_head_forward_residual: Z must not overlap H, W or R");
    hipStream_t st = static_cast<hipStream_t>(stream);
    const bool r_ok = R == nullptr || (reinterpret_cast<uintptr_t>(R) % 16 == 0 && ldr % 8 == 0);
    if (dt == BOM_BF16 && r_ok && bom::head_forward_stats_supported(H, ldh, W, ldw, Z, ldz, (int)N, (int)d, (int)V)) {
        hipError_t e = bom::launch_head_forward_stats(H, ldh, W, ldw, b, (int)N, (int)d, (int)V, Z, ldz, labels,
                                                      ignore_index, static_cast<float*>(workspace), row_target, st);
        if (e != hipSuccess) return hip_status(e, "bom_head_forward_residual (forward)");
        return hip_status(bom::launch_residual_from_stats(static_cast<const uint16_t*>(Z), ldz, (int)N, (int)V, labels,
                                                          ignore_index, s, row_lse, row_argmax, row_target,
                                                          static_cast<uint16_t*>(R), ldr, loss, n_valid, flags,
                                                          workspace, st),
                          "bom_head_forward_residual (residual)");
    }
    // other shapes and fp32: the forward, then the residual on its logits
    hipError_t e = bom::launch_head_forward(H, ldh, W, ldw, b, dt, (int)N, (int)d, (int)V, Z, ldz, st);
    if (e != hipSuccess) return hip_status(e, "bom_head_forward_residual (forward)");
    return hip_status(bom::launch_residual(Z, dt, (int)N, (int)V, ldz, labels, ignore_index, s, row_lse, row_argmax,
                                           row_target, R, ldr, loss, n_valid, flags, workspace, st),
                      "bom_head_forward_residual (residual)");
}

size_t bom_head_telemetry_workspace_bytes(int64_t N, int64_t d, int64_t V) {
    if (N < 1 || d < 1 || V < 1 || N >= kMaxDim || d >= kMaxDim || V >= kMaxDim) return 0;
    return bom::head_telemetry_workspace_bytes(N, d);
}

bom_status bom_head_telemetry(const void* H, int64_t ldh, bom_dtype h_dt, const void* R, int64_t ldr, bom_dtype r_dt,
                              int64_t N, int64_t d, int64_t V, const int32_t* labels, int32_t ignore_index,
                              const float* s, const float* q_hat, const int32_t* n_valid, float* M_W, int64_t ldm,
                              float* M_b, float beta1, int64_t t, float* out, void* workspace, size_t ws_bytes,
                              void* stream) {
    if (!H || !R || !labels || !s || !q_hat || !n_valid || !M_W || !out)
        return fail(BOM_ERR_NULL, "bom_head_telemetry: H, R, labels, s, q_hat, n_valid, M_W and out are required");
    if (N < 1 || d < 1 || V < 1 || N >= kMaxDim || d >= kMaxDim || V >= kMaxDim || ldh < d || ldr < V || ldm < V)
        return fail(BOM_ERR_SHAPE, "bom_head_telemetry: bad shape or leading dimension");
    if (!is_dtype(h_dt) || !is_dtype(r_dt)) return fail(BOM_ERR_DTYPE, "bom_head_telemetry: unsupported dtype");
    if (!(beta1 >= 0.f && beta1 < 1.f) || t < 1)
        return fail(BOM_ERR_HYPER, "bom_head_telemetry: need beta1 in [0, 1) and t >= 1");
    const size_t need = bom::head_telemetry_workspace_bytes(N, d);
    if (!workspace || ws_bytes < need)
        return fail(BOM_ERR_WORKSPACE, "bom_head_telemetry: workspace needs %zu bytes, got %zu", need, ws_bytes);
    if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
        return fail(BOM_ERR_WORKSPACE, "bom_head_telemetry: workspace must be 256-byte aligned");
    const size_t mb = ((size_t)(d - 1) * ldm + V) * 4;
    if ((M_b && overlap(M_W, mb, M_b, (size_t)V * 4)) || overlap(M_W, mb, out, 20) || (M_b && overlap(M_b, (size_t)V * 4, out, 20)))
        return fail(BOM_ERR_ALIAS, "bom_head_telemetry: M_W, M_b and out must be distinct");
    bom::TeleArgs a{H, ldh, h_dt, R, ldr, r_dt, (int)N, (int)d, (int)V, labels, ignore_index, s, q_hat, n_valid, M_W, ldm,
                    M_b, beta1, (float)(1.0 - (double)beta1),
                    (float)(1.0 / (1.0 - std::pow((double)beta1, (double)t))), out, workspace};
    return hip_status(bom::launch_head_telemetry(a, static_cast<hipStream_t>(stream)), "bom_head_telemetry");
}

bom_status bom_head_forward(const void* H, int64_t ldh, const void* W, int64_t ldw, const void* b, bom_dtype dt,
                            int64_t N, int64_t d, int64_t V, void* Z, int64_t ldz, void* stream) {
    if (!H || !W || !Z) return fail(BOM_ERR_NULL, "bom_head_forward: H, W and Z are required");
    if (N < 1 || d < 1 || V < 1 || N >= kMaxDim || d >= kMaxDim || V >= kMaxDim || ldh < d || ldw < V || ldz < V)
        return fail(BOM_ERR_SHAPE, "bom_head_forward: bad shape or leading dimension");
    if (!is_dtype(dt)) return fail(BOM_ERR_DTYPE, "bom_head_forward: unsupported dtype");
    if ((int64_t)N * V >= ((int64_t)1 << 40)) return fail(BOM_ERR_SHAPE, "bom_head_forward: output too large");
    return hip_status(bom::launch_head_forward(H, ldh, W, ldw, b, dt, (int)N, (int)d, (int)V, Z, ldz,
                                               static_cast<hipStream_t>(stream)),
                      "bom_head_forward");
}

}  // extern "C"
