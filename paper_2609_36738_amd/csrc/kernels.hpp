// Internal launch interface between the C-ABI layer (abi.hip) and the kernel files.
// Every launcher assumes its arguments were validated by the C-ABI layer.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "bom.h"

namespace bom {

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// ---- residual ------------------------------------------------------------------------------
size_t residual_workspace_bytes(int64_t N, int64_t V, bom_dtype dt);
hipError_t launch_residual(const void* Z, bom_dtype dt, int N, int V, int64_t ldz, const int32_t* labels,
                           int32_t ignore_index, float* s, float* row_lse, int32_t* row_argmax, float* row_target,
                           void* R, int64_t ldr, float* loss, int32_t* n_valid, int32_t* flags, void* ws,
                           hipStream_t stream);

// Allocation-free residual: the device address of this device's fixed scratch array (looked up once per
// device, with that device current) of kResidualScratchBytes, which takes the workspace's place.
constexpr size_t kResidualScratchBytes = (size_t)BOM_RESIDUAL_SCRATCH_BYTES;
hipError_t residual_scratch(void** ptr);

// ---- EMA -----------------------------------------------------------------------------------
hipError_t launch_ema(float* q, const float* s, int64_t V, float beta1, float inv_bc1, float* q_hat,
                      hipStream_t stream);

// ---- head VJP --------------------------------------------------------------------------------
struct HeadVjpArgs {
    const void* H; int64_t ldh;
    const void* W; int64_t ldw;
    const void* R; int64_t ldr;       // residual rows R, or the logits Z when is_residual == 0
    int is_residual;
    const float* row_lse;             // [N], read when is_residual == 0
    bom_dtype dt;
    int N, d, V;
    const int32_t* labels; int32_t ignore_index;
    const float* q_hat; const float* s; const int32_t* n_valid; float lambda;
    void* dW; bom_dtype dw_dt; int64_t lddw; float dW_beta;   // dW and db in dw_dt (fp32 or bf16)
    void* db;
    void* dH; bom_dtype dh_dt; int64_t lddh;
    void* ws; size_t ws_bytes;
};
size_t head_vjp_workspace_bytes(int64_t N, int64_t d, int64_t V, bom_dtype dt, bom_dtype dw_dt);
hipError_t launch_head_vjp(const HeadVjpArgs& a, hipStream_t stream);

// ---- head telemetry (diagnostic) --------------------------------------------------------------
struct TeleArgs {
    const void* H; int64_t ldh; bom_dtype h_dt;
    const void* R; int64_t ldr; bom_dtype r_dt;
    int N, d, V;
    const int32_t* labels; int32_t ignore_index;
    const float* s; const float* q_hat; const int32_t* n_valid;
    float* MW; int64_t ldm; float* Mb;
    float beta1, one_minus_beta1, inv_bc;
    float* out;
    void* ws;
};
size_t head_telemetry_workspace_bytes(int64_t N, int64_t d);
hipError_t launch_head_telemetry(const TeleArgs& a, hipStream_t stream);

// ---- head forward (support) ---------------------------------------------------------------
hipError_t launch_head_forward(const void* H, int64_t ldh, const void* W, int64_t ldw, const void* b, bom_dtype dt,
                               int N, int d, int V, void* Z, int64_t ldz, hipStream_t stream);

// ---- head forward with row statistics, then the residual from them --------------------------------
// The forward on the 256-tile MFMA kernel also writes, per row and 256-column tile, (max, sum of
// exp(z - max), first argmax) of the rounded logits ([N][ceil(V/256)][3] floats) and the target logit of
// each row whose label is valid. Unsupported shapes (see head_forward_stats_supported) return
// hipErrorInvalidValue.
bool head_forward_stats_supported(const void* H, int64_t ldh, const void* W, int64_t ldw, const void* Z, int64_t ldz,
                                  int N, int d, int V);
hipError_t launch_head_forward_stats(const void* H, int64_t ldh, const void* W, int64_t ldw, const void* b, int N, int d,
                                     int V, void* Z, int64_t ldz, const int32_t* labels, int32_t ignore_index,
                                     float* stats, float* row_target, hipStream_t stream);
size_t residual_from_stats_workspace_bytes(int64_t N, int64_t V);
hipError_t launch_residual_from_stats(const uint16_t* Z, int64_t ldz, int N, int V, const int32_t* labels,
                                      int32_t ignore_index, float* s, float* row_lse, int32_t* row_argmax,
                                      float* row_target, uint16_t* R, int64_t ldr, float* loss, int32_t* n_valid,
                                      int32_t* flags, void* ws, hipStream_t stream);

// ---- update ----------------------------------------------------------------------------------
struct SegTable {
    int n;
    int64_t begin[BOM_MAX_SEGMENTS];
    int64_t end[BOM_MAX_SEGMENTS];
    float wd[BOM_MAX_SEGMENTS];
    float wd_default;
};
struct UpdateScalars {
    float lr, beta2, one_minus_beta2, eps, lambda, u_scale, inv_bc2;
    float clip_norm;      // > 0: global-norm clipping of the numerator
    const float* clip;    // device word with the clipping factor (written on the device), or null
    float* clip_stats;    // optional device [2]: the numerator's norm before clipping and the factor
    float beta1, one_minus_beta1, inv_bc1;   // AdamW's first moment (the comparison update)
};
size_t update_workspace_bytes(int64_t P, const bom_update_cfg* cfg);
hipError_t launch_update_dense(float* theta, float* v, const float* u, const float* h, int64_t P, const SegTable& segs,
                               UpdateScalars sc, void* ws, hipStream_t stream);
hipError_t launch_update_dense_bf16(uint16_t* theta, uint16_t* v, const uint16_t* u, const uint16_t* h, int64_t P,
                                    const SegTable& segs, UpdateScalars sc, void* ws, hipStream_t stream);
// Block-shared second moment: segments tiling [0, P) in order, each cut into blocks of blk[k] elements.
struct BlockSegs {
    int n;
    int64_t begin[BOM_MAX_SEGMENTS];
    int64_t len[BOM_MAX_SEGMENTS];
    int64_t blk[BOM_MAX_SEGMENTS];
    float wd[BOM_MAX_SEGMENTS];
};
int64_t blocks_count(const BlockSegs& b);
hipError_t launch_update_blocks(float* theta, float* v, const float* u, const float* h, int64_t P, const BlockSegs& bs,
                                UpdateScalars sc, void* ws, hipStream_t stream);
hipError_t launch_update_factored(float* theta, float* Rr, float* Cc, const float* u, const float* h, int64_t P,
                                  int64_t block_rows, int64_t block_cols, const SegTable& segs,
                                  const UpdateScalars& sc, void* ws, hipStream_t stream);
// AdamW (the comparison optimizer of the cost model): dense, or with the factored second moment for
// block_cols of 1024, 2048 or 4096.
hipError_t launch_adamw_dense(float* theta, float* m, float* v, const float* g, int64_t P, const SegTable& segs,
                              const UpdateScalars& sc, hipStream_t stream);
hipError_t launch_adamw_factored(float* theta, float* m, float* Rr, float* Cc, const float* g, int64_t P,
                                 int64_t block_rows, int64_t block_cols, const SegTable& segs, const UpdateScalars& sc,
                                 void* ws, hipStream_t stream);

}  // namespace bom
