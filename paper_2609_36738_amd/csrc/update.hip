// bom_update kernels: second moment of the BOM numerator and the decoupled-decay update over one
// flat fp32 parameter buffer (Sec. 3.4; Algorithm 1, the second-moment and parameter updates). There is no first
// moment: 20 bytes per parameter (read theta, v, u; write theta, v), 24 with a split numerator.
//
// Factored layout (a reading; the paper does not define one): the buffer is a row-major matrix of
// block_cols columns grouped into blocks of block_rows rows; v_hat_ij = Rr_i Cc_j / sum(Rr) / bc2.
// Three launches: row/column statistics of u'^2 (one read of u), a per-block finish (Cc and the
// block sum of Rr), and the parameter update (one more read of u, read + write of theta).
//
// Block-shared layout (Adam-mini's map with the BOM numerator): one v per block of consecutive parameters,
// block lengths per segment. Blocks of up to 4096 elements: one wave per block keeps the block in
// registers between its statistics and its step (read u and theta, write theta: 12 bytes per parameter).
// Longer blocks: pieces of 4096 elements, one wave each, for fp32 partial sums, a per-block finish in piece
// order, and the step (16 bytes per parameter). Blocks of one element take the dense kernels.
//
// Global-norm clipping (clip_norm > 0): u' is scaled by c = min(1, clip_norm / (||u'|| + 1e-6)), the
// norm over the whole buffer, computed on the device. Dense layout: one extra read of the numerator
// (per-workgroup fp64 partial sums, one finishing workgroup). Factored layout: no extra pass over u;
// the statistics kernel keeps the row sums rho_i of u'^2 unclipped, their total is ||u'||^2, and
// the finish kernels fold c^2 into the updates of Rr and Cc before the parameter step uses c u'.
#include "common.hpp"
#include "kernels.hpp"

namespace bom {
namespace {

constexpr int kUpdThreads = 256;
constexpr int kFacRowsPerWG = 64;   // rows of u per statistics workgroup (inside one block)
constexpr int kFacUpdRows = 8;      // rows per update workgroup

__device__ __forceinline__ float decay_of(int64_t e, const SegTable& t) {
    float wd = t.wd_default;
    for (int k = t.n - 1; k >= 0; --k)
        if (e >= t.begin[k] && e < t.end[k]) wd = t.wd[k];
    return wd;
}

template <bool SPLIT>
__device__ __forceinline__ float numerator(float u, float h, const UpdateScalars& sc) {
    if (SPLIT) return sc.u_scale * ((1.0f - sc.lambda) * u + sc.lambda * h);
    return sc.u_scale * u;
}

// The scalars of a parameter step: u_scale times the clipping factor when clipping is on.
__device__ __forceinline__ UpdateScalars clipped(UpdateScalars sc) {
    if (sc.clip) sc.u_scale *= *sc.clip;
    return sc;
}

__device__ __forceinline__ void adam_style(float& th, float& v, float up, float wd, const UpdateScalars& sc) {
    v = sc.beta2 * v + sc.one_minus_beta2 * (up * up);
    const float vhat = v * sc.inv_bc2;
    th = (1.0f - sc.lr * wd) * th - sc.lr * (up / (sqrtf(vhat) + sc.eps));
}

// ---- dense ----------------------------------------------------------------------------------
// One launch over [0, P): elements [0, head) and the tail past head + 4 nvec one per thread (threads
// nvec, nvec + 1, ... of the grid), the body [head, head + 4 nvec) one 16-byte group per thread, with
// non-temporal loads and stores (each byte is touched once). head makes theta + head, v + head,
// u + head (and h + head) 16-byte aligned: the arrays share their offset inside a 16-byte group.
template <bool SPLIT>
__global__ __launch_bounds__(kUpdThreads) void update_dense_vec4_kernel(float* __restrict__ theta, float* __restrict__ v,
                                                                        const float* __restrict__ u,
                                                                        const float* __restrict__ h, int64_t head,
                                                                        int64_t nvec, int64_t P, SegTable segs,
                                                                        UpdateScalars sc) {
    const int64_t q = (int64_t)blockIdx.x * kUpdThreads + threadIdx.x;
    sc = clipped(sc);
    if (q >= nvec) {
        const int64_t r = q - nvec;
        const int64_t tail0 = head + 4 * nvec;
        const int64_t e = r < head ? r : tail0 + (r - head);
        if (e >= P) return;
        float t = theta[e], vv = v[e];
        adam_style(t, vv, numerator<SPLIT>(u[e], SPLIT ? h[e] : 0.f, sc), decay_of(e, segs), sc);
        theta[e] = t;
        v[e] = vv;
        return;
    }
    const int64_t e = head + q * 4;
    f32x4 t4 = ld_stream(theta + e);
    f32x4 v4 = ld_stream(v + e);
    const f32x4 u4 = ld_stream(u + e);
    f32x4 h4 = {0.f, 0.f, 0.f, 0.f};
    if (SPLIT) h4 = ld_stream(h + e);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        float th = t4[c], vv = v4[c];
        adam_style(th, vv, numerator<SPLIT>(u4[c], h4[c], sc), decay_of(e + c, segs), sc);
        t4[c] = th;
        v4[c] = vv;
    }
    st_stream(theta + e, t4);
    st_stream(v + e, v4);
}

template <bool SPLIT>
__global__ __launch_bounds__(kUpdThreads) void update_dense_scalar_kernel(float* __restrict__ theta, float* __restrict__ v,
                                                                          const float* __restrict__ u,
                                                                          const float* __restrict__ h, int64_t begin,
                                                                          int64_t end, SegTable segs, UpdateScalars sc) {
    const int64_t stride = (int64_t)gridDim.x * kUpdThreads;
    sc = clipped(sc);
    for (int64_t e = begin + (int64_t)blockIdx.x * kUpdThreads + threadIdx.x; e < end; e += stride) {
        float t = theta[e], vv = v[e];
        adam_style(t, vv, numerator<SPLIT>(u[e], SPLIT ? h[e] : 0.f, sc), decay_of(e, segs), sc);
        theta[e] = t;
        v[e] = vv;
    }
}

// ---- AdamW (the comparison arm of the cost model) ---------------------------------------------------
// The dense first moment BOM deletes: m = b1 m + (1 - b1) g, v = b2 v + (1 - b2) g^2,
// theta = (1 - lr w) theta - lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps); 28 bytes per parameter.
__device__ __forceinline__ void adamw_step(float& th, float& m, float& v, float g, float wd, const UpdateScalars& sc) {
    m = sc.beta1 * m + sc.one_minus_beta1 * g;
    v = sc.beta2 * v + sc.one_minus_beta2 * (g * g);
    const float vhat = v * sc.inv_bc2;
    th = (1.0f - sc.lr * wd) * th - sc.lr * ((m * sc.inv_bc1) / (sqrtf(vhat) + sc.eps));
}

// One launch over [0, P) laid out like update_dense_vec4_kernel: scalar head and tail, 16-byte groups.
__global__ __launch_bounds__(kUpdThreads) void adamw_dense_vec4_kernel(float* __restrict__ theta, float* __restrict__ m,
                                                                       float* __restrict__ v, const float* __restrict__ g,
                                                                       int64_t head, int64_t nvec, int64_t P,
                                                                       SegTable segs, UpdateScalars sc) {
    const int64_t q = (int64_t)blockIdx.x * kUpdThreads + threadIdx.x;
    if (q >= nvec) {
        const int64_t r = q - nvec;
        const int64_t e = r < head ? r : head + 4 * nvec + (r - head);
        if (e >= P) return;
        float t = theta[e], mm = m[e], vv = v[e];
        adamw_step(t, mm, vv, sc.u_scale * g[e], decay_of(e, segs), sc);
        theta[e] = t;
        m[e] = mm;
        v[e] = vv;
        return;
    }
    const int64_t e = head + q * 4;
    f32x4 t4 = ld_stream(theta + e);
    f32x4 m4 = ld_stream(m + e);
    f32x4 v4 = ld_stream(v + e);
    const f32x4 g4 = ld_stream(g + e);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        float th = t4[c], mm = m4[c], vv = v4[c];
        adamw_step(th, mm, vv, sc.u_scale * g4[c], decay_of(e + c, segs), sc);
        t4[c] = th;
        m4[c] = mm;
        v4[c] = vv;
    }
    st_stream(theta + e, t4);
    st_stream(m + e, m4);
    st_stream(v + e, v4);
}

__global__ __launch_bounds__(kUpdThreads) void adamw_dense_scalar_kernel(float* __restrict__ theta, float* __restrict__ m,
                                                                         float* __restrict__ v,
                                                                         const float* __restrict__ g, int64_t P,
                                                                         SegTable segs, UpdateScalars sc) {
    const int64_t stride = (int64_t)gridDim.x * kUpdThreads;
    for (int64_t e = (int64_t)blockIdx.x * kUpdThreads + threadIdx.x; e < P; e += stride) {
        float t = theta[e], mm = m[e], vv = v[e];
        adamw_step(t, mm, vv, sc.u_scale * g[e], decay_of(e, segs), sc);
        theta[e] = t;
        m[e] = mm;
        v[e] = vv;
    }
}

// ---- dense, bf16 storage ------------------------------------------------------------------------
// theta, v, u (and h) stored as bf16 (10 bytes per parameter, 12 with h); the step is computed in fp32
// from the widened values and theta and v are rounded to nearest-even bf16 when stored. Eight elements
// (16 bytes of each array) per thread.
__device__ __forceinline__ float bf16_at(const u32x4_t& x, int c) { return c & 1 ? bf16_hi(x[c / 2]) : bf16_lo(x[c / 2]); }

// One launch over [0, P) like the fp32 kernel: scalar head and tail, 16-byte groups of 8 in between.
template <bool SPLIT>
__global__ __launch_bounds__(kUpdThreads) void update_dense_bf16x8_kernel(uint16_t* __restrict__ theta,
                                                                          uint16_t* __restrict__ v,
                                                                          const uint16_t* __restrict__ u,
                                                                          const uint16_t* __restrict__ h, int64_t head,
                                                                          int64_t nvec, int64_t P, SegTable segs,
                                                                          UpdateScalars sc) {
    const int64_t q = (int64_t)blockIdx.x * kUpdThreads + threadIdx.x;
    sc = clipped(sc);
    if (q >= nvec) {
        const int64_t r = q - nvec;
        const int64_t tail0 = head + 8 * nvec;
        const int64_t e = r < head ? r : tail0 + (r - head);
        if (e >= P) return;
        float t = bf16_to_f32(theta[e]), vv = bf16_to_f32(v[e]);
        adam_style(t, vv, numerator<SPLIT>(bf16_to_f32(u[e]), SPLIT ? bf16_to_f32(h[e]) : 0.f, sc), decay_of(e, segs), sc);
        theta[e] = f32_to_bf16(t);
        v[e] = f32_to_bf16(vv);
        return;
    }
    const int64_t e = head + q * 8;
    const u32x4_t t8 = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(theta + e));
    const u32x4_t v8 = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(v + e));
    const u32x4_t u8 = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(u + e));
    u32x4_t h8 = {0u, 0u, 0u, 0u};
    if (SPLIT) h8 = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(h + e));
    float th[8], vv[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        th[c] = bf16_at(t8, c);
        vv[c] = bf16_at(v8, c);
        adam_style(th[c], vv[c], numerator<SPLIT>(bf16_at(u8, c), SPLIT ? bf16_at(h8, c) : 0.f, sc), decay_of(e + c, segs),
                   sc);
    }
    u32x4_t to, vo;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        to[k] = pack_bf16x2(th[2 * k], th[2 * k + 1]);
        vo[k] = pack_bf16x2(vv[2 * k], vv[2 * k + 1]);
    }
    __builtin_nontemporal_store(to, reinterpret_cast<u32x4_t*>(theta + e));
    __builtin_nontemporal_store(vo, reinterpret_cast<u32x4_t*>(v + e));
}

template <bool SPLIT>
__global__ __launch_bounds__(kUpdThreads) void update_dense_bf16_scalar_kernel(uint16_t* __restrict__ theta,
                                                                               uint16_t* __restrict__ v,
                                                                               const uint16_t* __restrict__ u,
                                                                               const uint16_t* __restrict__ h,
                                                                               int64_t begin, int64_t end, SegTable segs,
                                                                               UpdateScalars sc) {
    const int64_t stride = (int64_t)gridDim.x * kUpdThreads;
    sc = clipped(sc);
    for (int64_t e = begin + (int64_t)blockIdx.x * kUpdThreads + threadIdx.x; e < end; e += stride) {
        float t = bf16_to_f32(theta[e]), vv = bf16_to_f32(v[e]);
        adam_style(t, vv, numerator<SPLIT>(bf16_to_f32(u[e]), SPLIT ? bf16_to_f32(h[e]) : 0.f, sc), decay_of(e, segs), sc);
        theta[e] = f32_to_bf16(t);
        v[e] = f32_to_bf16(vv);
    }
}

// ---- factored --------------------------------------------------------------------------------
// Statistics: workgroup w covers rows [r0, r1) of one block; thread t owns columns (k*256 + t)*4..+3.
template <bool SPLIT, int KC>
__global__ __launch_bounds__(kUpdThreads) void factored_stats_kernel(const float* __restrict__ u,
                                                                     const float* __restrict__ h, int64_t P,
                                                                     int64_t nrows, int64_t block_rows, int bc,
                                                                     int groups_per_block, float* __restrict__ Rr,
                                                                     float* __restrict__ kpart, float* __restrict__ rho_out,
                                                                     UpdateScalars sc) {
    __shared__ float sh[kUpdThreads / kWave];
    const int t = threadIdx.x;
    const int64_t b = blockIdx.x / groups_per_block;
    const int64_t g = blockIdx.x % groups_per_block;
    const int64_t blk_end = min((b + 1) * block_rows, nrows);
    const int64_t r0 = b * block_rows + g * kFacRowsPerWG;
    const int64_t r1 = min(r0 + kFacRowsPerWG, blk_end);
    float kap[KC * 4];
#pragma unroll
    for (int k = 0; k < KC * 4; ++k) kap[k] = 0.f;
    for (int64_t i = r0; i < r1; ++i) {
        float rho = 0.f;
#pragma unroll
        for (int k = 0; k < KC; ++k) {
            const int j = (k * kUpdThreads + t) * 4;
            const int64_t e = i * bc + j;
            if (j < bc && e < P) {
                const f32x4 u4 = ld_stream(u + e);
                f32x4 h4 = {0.f, 0.f, 0.f, 0.f};
                if (SPLIT) h4 = ld_stream(h + e);
                const float a0 = numerator<SPLIT>(u4[0], h4[0], sc), a1 = numerator<SPLIT>(u4[1], h4[1], sc);
                const float a2 = numerator<SPLIT>(u4[2], h4[2], sc), a3 = numerator<SPLIT>(u4[3], h4[3], sc);
                const float s0 = a0 * a0, s1 = a1 * a1, s2 = a2 * a2, s3 = a3 * a3;
                kap[k * 4 + 0] += s0;
                kap[k * 4 + 1] += s1;
                kap[k * 4 + 2] += s2;
                kap[k * 4 + 3] += s3;
                rho += (s0 + s1) + (s2 + s3);
            }
        }
        rho = wave_sum(rho);
        if ((t & (kWave - 1)) == 0) sh[t / kWave] = rho;
        __syncthreads();
        if (t == 0) {
            float r = 0.f;
#pragma unroll
            for (int w = 0; w < kUpdThreads / kWave; ++w) r += sh[w];
            if (rho_out) rho_out[i] = r;   // clipping: Rr is updated once the factor is known
            else Rr[i] = sc.beta2 * Rr[i] + sc.one_minus_beta2 * r;
        }
        __syncthreads();
    }
    float* kp = kpart + (int64_t)blockIdx.x * bc;
#pragma unroll
    for (int k = 0; k < KC; ++k) {
        const int j = (k * kUpdThreads + t) * 4;
        if (j < bc) *reinterpret_cast<float4*>(kp + j) = make_float4(kap[k * 4], kap[k * 4 + 1], kap[k * 4 + 2], kap[k * 4 + 3]);
    }
}

// Per-block finish: Cc_j = beta2 Cc_j + (1-beta2) sum_g kpart[g][j]; rsum[b] = sum of the block's Rr.
__global__ __launch_bounds__(kUpdThreads) void factored_finish_kernel(const float* __restrict__ kpart,
                                                                      int groups_per_block, int64_t nrows,
                                                                      int64_t block_rows, int bc, float* __restrict__ Rr,
                                                                      float* __restrict__ Cc, float* __restrict__ rsum,
                                                                      const float* __restrict__ rho, UpdateScalars sc) {
    const float c2 = rho ? *sc.clip * *sc.clip : 1.f;   // clipping scales u'^2 by c^2
    __shared__ float sh[kUpdThreads];
    const int64_t b = blockIdx.x;
    const int t = threadIdx.x;
    const int64_t r0 = b * block_rows;
    const int64_t r1 = min(r0 + block_rows, nrows);
    const int ng = (int)((r1 - r0 + kFacRowsPerWG - 1) / kFacRowsPerWG);
    const float* kp = kpart + b * groups_per_block * (int64_t)bc;
    for (int j = t; j < bc; j += kUpdThreads) {
        float c = 0.f;
        for (int g = 0; g < ng; ++g) c += kp[(int64_t)g * bc + j];
        Cc[b * bc + j] = sc.beta2 * Cc[b * bc + j] + sc.one_minus_beta2 * (c2 * c);
    }
    float r = 0.f;
    for (int64_t i = r0 + t; i < r1; i += kUpdThreads) {
        if (rho) Rr[i] = sc.beta2 * Rr[i] + sc.one_minus_beta2 * (c2 * rho[i]);
        r += Rr[i];
    }
    sh[t] = r;
    __syncthreads();
    for (int o = kUpdThreads / 2; o > 0; o >>= 1) {
        if (t < o) sh[t] += sh[t + o];
        __syncthreads();
    }
    if (t == 0) rsum[b] = sh[0];
}

// Update: workgroup covers kFacUpdRows rows; v_hat_ij = (Rr_i / rsum_b * inv_bc2) * Cc_j. theta and u
// are streamed (non-temporal, each byte touched once); the small Cc stays cached for the block's rows.
template <bool SPLIT, int KC>
__global__ __launch_bounds__(kUpdThreads) void factored_update_kernel(float* __restrict__ theta, const float* __restrict__ u,
                                                                      const float* __restrict__ h, int64_t P, int64_t nrows,
                                                                      int64_t block_rows, int bc,
                                                                      const float* __restrict__ Rr,
                                                                      const float* __restrict__ Cc,
                                                                      const float* __restrict__ rsum, SegTable segs,
                                                                      UpdateScalars sc) {
    const int t = threadIdx.x;
    sc = clipped(sc);
    const int64_t r0 = (int64_t)blockIdx.x * kFacUpdRows;
    const int64_t r1 = min(r0 + kFacUpdRows, nrows);
    for (int64_t i = r0; i < r1; ++i) {
        const int64_t b = i / block_rows;
        const float rs = rsum[b];
        const float a = rs > 0.f ? Rr[i] / rs * sc.inv_bc2 : 0.f;
        const float* cb = Cc + b * bc;
        f32x4 t4[KC], u4[KC], h4[KC], c4[KC];
#pragma unroll
        for (int k = 0; k < KC; ++k) {   // clamped loads, all in flight; stores below are guarded
            const int j = (k * kUpdThreads + t) * 4;
            const int jc = j < bc ? j : bc - 4;
            const int64_t e = i * bc + jc;
            const int64_t ec = e < P ? e : P - 4;
            t4[k] = ld_stream(theta + ec);
            u4[k] = ld_stream(u + ec);
            if (SPLIT) h4[k] = ld_stream(h + ec);
            c4[k] = *reinterpret_cast<const f32x4*>(cb + jc);
        }
#pragma unroll
        for (int k = 0; k < KC; ++k) {
            const int j = (k * kUpdThreads + t) * 4;
            const int64_t e = i * bc + j;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const float up = numerator<SPLIT>(u4[k][c], SPLIT ? h4[k][c] : 0.f, sc);
                const float vhat = a * c4[k][c];
                const float wd = decay_of(e + c, segs);
                t4[k][c] = (1.0f - sc.lr * wd) * t4[k][c] - sc.lr * (up / (sqrtf(vhat) + sc.eps));
            }
            if (j < bc && e < P) st_stream(theta + e, t4[k]);
        }
    }
}

// Update for block_cols = NV * 256: one workgroup per row i (a scalar, like its block b = i / block_rows
// and the row scale Rr_i / rsum_b / bc2), thread t holding columns (k*256 + t)*4 .. +3 for k < NV/4, so
// no per-element index arithmetic and NV/4 16-byte loads of theta and of u in flight per thread.
// Elements at or past P (only in the last row) are loaded from a clamped address and not stored.
template <bool SPLIT, int NV>
__global__ __launch_bounds__(kUpdThreads) void factored_update_rows_kernel(float* __restrict__ theta,
                                                                          const float* __restrict__ u,
                                                                          const float* __restrict__ h, int64_t P,
                                                                          int64_t block_rows,
                                                                          const float* __restrict__ Rr,
                                                                          const float* __restrict__ Cc,
                                                                          const float* __restrict__ rsum, SegTable segs,
                                                                          UpdateScalars sc) {
    constexpr int BC = NV * 256;
    constexpr int KV = NV / 4;   // 16-byte groups per thread
    const int64_t i = blockIdx.x;
    sc = clipped(sc);
    const int64_t b = i / block_rows;
    const float rs = rsum[b];
    const float a = rs > 0.f ? Rr[i] / rs * sc.inv_bc2 : 0.f;
    const float* cb = Cc + b * BC;
    const int t = threadIdx.x;
    f32x4 t4[KV], u4[KV], h4[KV], c4[KV];
#pragma unroll
    for (int k = 0; k < KV; ++k) {
        const int j = (k * kUpdThreads + t) * 4;
        const int64_t e = i * BC + j;
        const int64_t ec = e < P ? e : P - 4;
        t4[k] = ld_stream(theta + ec);
        u4[k] = ld_stream(u + ec);
        if (SPLIT) h4[k] = ld_stream(h + ec);
        c4[k] = *reinterpret_cast<const f32x4*>(cb + j);
    }
#pragma unroll
    for (int k = 0; k < KV; ++k) {
        const int j = (k * kUpdThreads + t) * 4;
        const int64_t e = i * BC + j;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const float up = numerator<SPLIT>(u4[k][c], SPLIT ? h4[k][c] : 0.f, sc);
            const float vhat = a * c4[k][c];
            t4[k][c] = (1.0f - sc.lr * decay_of(e + c, segs)) * t4[k][c] - sc.lr * (up / (sqrtf(vhat) + sc.eps));
        }
        if (e < P) st_stream(theta + e, t4[k]);
    }
}

// Row kernels for block_cols = NV * 256 (up to 4096): a wave owns whole rows, lane l holding
// columns (k*64 + l)*4 .. +3 for k < NV, so each row's loads are all in flight together and the row
// statistic is one wave reduction. Elements at or past P (only in the last row) count as zero. The
// statistics read u with non-temporal loads (8B parameters: 5.73 -> 5.22 ms against cached loads).
// AdamW with the factored second moment (block_cols = NV * 256): the update of factored_update_rows_kernel
// with the numerator m_hat, m = b1 m + (1 - b1) g read and written in the same pass.
template <int NV>
__global__ __launch_bounds__(kUpdThreads) void factored_adamw_rows_kernel(float* __restrict__ theta, float* __restrict__ m,
                                                                          const float* __restrict__ g, int64_t P,
                                                                          int64_t block_rows,
                                                                          const float* __restrict__ Rr,
                                                                          const float* __restrict__ Cc,
                                                                          const float* __restrict__ rsum, SegTable segs,
                                                                          UpdateScalars sc) {
    constexpr int BC = NV * 256;
    constexpr int KV = NV / 4;
    const int64_t i = blockIdx.x;
    const int64_t b = i / block_rows;
    const float rs = rsum[b];
    const float a = rs > 0.f ? Rr[i] / rs * sc.inv_bc2 : 0.f;
    const float* cb = Cc + b * BC;
    const int t = threadIdx.x;
    f32x4 t4[KV], g4[KV], m4[KV], c4[KV];
#pragma unroll
    for (int k = 0; k < KV; ++k) {
        const int j = (k * kUpdThreads + t) * 4;
        const int64_t e = i * BC + j;
        const int64_t ec = e < P ? e : P - 4;
        t4[k] = ld_stream(theta + ec);
        g4[k] = ld_stream(g + ec);
        m4[k] = ld_stream(m + ec);
        c4[k] = *reinterpret_cast<const f32x4*>(cb + j);
    }
#pragma unroll
    for (int k = 0; k < KV; ++k) {
        const int j = (k * kUpdThreads + t) * 4;
        const int64_t e = i * BC + j;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const float mm = sc.beta1 * m4[k][c] + sc.one_minus_beta1 * (sc.u_scale * g4[k][c]);
            const float vhat = a * c4[k][c];
            m4[k][c] = mm;
            t4[k][c] = (1.0f - sc.lr * decay_of(e + c, segs)) * t4[k][c] - sc.lr * ((mm * sc.inv_bc1) / (sqrtf(vhat) + sc.eps));
        }
        if (e < P) {
            st_stream(theta + e, t4[k]);
            st_stream(m + e, m4[k]);
        }
    }
}

template <bool SPLIT, int NV>
__global__ __launch_bounds__(kUpdThreads) void factored_stats_rows_kernel(const float* __restrict__ u,
                                                                          const float* __restrict__ h, int64_t P,
                                                                          int64_t nrows, int64_t block_rows,
                                                                          int groups_per_block, float* __restrict__ Rr,
                                                                          float* __restrict__ kpart,
                                                                          float* __restrict__ rho_out, UpdateScalars sc) {
    constexpr int BC = NV * 256;
    __shared__ f32x4 sh[3][BC / 4];
    const int t = threadIdx.x, l = t % kWave, w = t / kWave;
    const int64_t b = blockIdx.x / groups_per_block;
    const int64_t g = blockIdx.x % groups_per_block;
    const int64_t blk_end = min((b + 1) * block_rows, nrows);
    const int64_t r0 = b * block_rows + g * kFacRowsPerWG;
    const int64_t r1 = min(r0 + kFacRowsPerWG, blk_end);
    f32x4 kap[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k) kap[k] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int64_t i = r0 + w; i < r1; i += kUpdThreads / kWave) {
        f32x4 a[NV];
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            const int64_t e = i * BC + (k * kWave + l) * 4;
            const bool ok = e < P;
            const int64_t ec = ok ? e : P - 4;
            const f32x4 u4 = ld_stream(u + ec);
            f32x4 h4 = {0.f, 0.f, 0.f, 0.f};
            if (SPLIT) h4 = ld_stream(h + ec);
            const float z = ok ? 1.f : 0.f;
#pragma unroll
            for (int c = 0; c < 4; ++c) a[k][c] = z * numerator<SPLIT>(u4[c], h4[c], sc);
        }
        float rho = 0.f;
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            const f32x4 s2 = a[k] * a[k];
            kap[k] += s2;
            rho += (s2[0] + s2[1]) + (s2[2] + s2[3]);
        }
        rho = wave_sum(rho);
        if (l == 0) {
            if (rho_out) rho_out[i] = rho;   // clipping: Rr is updated once the factor is known
            else Rr[i] = sc.beta2 * Rr[i] + sc.one_minus_beta2 * rho;
        }
    }
    if (w > 0) {
#pragma unroll
        for (int k = 0; k < NV; ++k) sh[w - 1][k * kWave + l] = kap[k];
    }
    __syncthreads();
    if (w == 0) {
        float* kp = kpart + (int64_t)blockIdx.x * BC;
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            const int q = k * kWave + l;
            *reinterpret_cast<f32x4*>(kp + q * 4) = ((kap[k] + sh[0][q]) + sh[1][q]) + sh[2][q];
        }
    }
}

// Per-block finish over column chunks of 1024: Cc_j = beta2 Cc_j + (1 - beta2) sum_g kpart[g][j] (in
// group order); chunk 0 also forms rsum[b] = sum of the block's Rr.
__global__ __launch_bounds__(kUpdThreads) void factored_finish_cols_kernel(const float* __restrict__ kpart,
                                                                           int groups_per_block, int64_t nrows,
                                                                           int64_t block_rows, int bc, int nchunks,
                                                                           float* __restrict__ Rr,
                                                                           float* __restrict__ Cc,
                                                                           float* __restrict__ rsum,
                                                                           const float* __restrict__ rho, UpdateScalars sc) {
    __shared__ float sh[kUpdThreads];
    const float c2 = rho ? *sc.clip * *sc.clip : 1.f;   // clipping scales u'^2 by c^2
    const int64_t b = blockIdx.x / nchunks;
    const int chunk = blockIdx.x % nchunks;
    const int t = threadIdx.x;
    const int64_t r0 = b * block_rows;
    const int64_t r1 = min(r0 + block_rows, nrows);
    const int ng = (int)((r1 - r0 + kFacRowsPerWG - 1) / kFacRowsPerWG);
    const float* kp = kpart + b * groups_per_block * (int64_t)bc;
    const int j = chunk * 1024 + t * 4;
    if (j < bc) {
        f32x4 c = {0.f, 0.f, 0.f, 0.f};
        int gi = 0;
        for (; gi + 4 <= ng; gi += 4) {
            const f32x4 p0 = *reinterpret_cast<const f32x4*>(kp + (int64_t)(gi + 0) * bc + j);
            const f32x4 p1 = *reinterpret_cast<const f32x4*>(kp + (int64_t)(gi + 1) * bc + j);
            const f32x4 p2 = *reinterpret_cast<const f32x4*>(kp + (int64_t)(gi + 2) * bc + j);
            const f32x4 p3 = *reinterpret_cast<const f32x4*>(kp + (int64_t)(gi + 3) * bc + j);
            c += p0;
            c += p1;
            c += p2;
            c += p3;
        }
        for (; gi < ng; ++gi) c += *reinterpret_cast<const f32x4*>(kp + (int64_t)gi * bc + j);
        f32x4 old = *reinterpret_cast<const f32x4*>(Cc + b * bc + j);
        *reinterpret_cast<f32x4*>(Cc + b * bc + j) = sc.beta2 * old + sc.one_minus_beta2 * (c2 * c);
    }
    if (chunk != 0) return;
    float r = 0.f;
    for (int64_t i = r0 + t; i < r1; i += kUpdThreads) {
        if (rho) Rr[i] = sc.beta2 * Rr[i] + sc.one_minus_beta2 * (c2 * rho[i]);
        r += Rr[i];
    }
    sh[t] = r;
    __syncthreads();
    for (int o = kUpdThreads / 2; o > 0; o >>= 1) {
        if (t < o) sh[t] += sh[t + o];
        __syncthreads();
    }
    if (t == 0) rsum[b] = sh[0];
}

// ---- global-norm clipping ------------------------------------------------------------------
// ---- block-shared second moment ------------------------------------------------------------------
// Pointers are at the segment's first element (theta, u, h) and first block (v); len elements, blocks of
// blk (the last one may be shorter), nblk = ceil(len / blk). VEC: 16-byte accesses (the host checks that
// the segment's pointers are 16-byte aligned and that blk and len are multiples of 4).
constexpr int kBlkWave = 4096;                       // longest block held by one wave
constexpr int kWavesPerWG = kUpdThreads / kWave;
// partial sums of blocks longer than kBlkWave: a segment of n elements cut into blocks of blk > kBlkWave
// (blk at most n) has ceil(n / blk) ceil(blk / kBlkWave) <= 3 n / kBlkWave + 1 pieces
size_t blocks_part_bytes(int64_t P) { return align256((size_t)(P / 1024 + 64) * sizeof(float)); }

template <bool SPLIT, int NV, bool VEC>
__global__ __launch_bounds__(kUpdThreads) void blocks_wave_kernel(float* __restrict__ theta, float* __restrict__ v,
                                                                  const float* __restrict__ u,
                                                                  const float* __restrict__ h, int64_t len,
                                                                  int64_t blk, int64_t nblk, float wd, UpdateScalars sc) {
    const int lane = threadIdx.x % kWave;
    const int64_t b = (int64_t)blockIdx.x * kWavesPerWG + threadIdx.x / kWave;
    if (b >= nblk) return;   // the whole wave
    sc = clipped(sc);
    const int64_t e0 = b * blk;
    const int n = (int)(blk < len - e0 ? blk : len - e0);
    float up[4 * NV], th[4 * NV];
    float ss = 0.f;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        if constexpr (VEC) {
            const int j = (lane + kWave * k) * 4;
            if (j < n) {
                const f32x4 u4 = ld_stream(u + e0 + j);
                const f32x4 t4 = ld_stream(theta + e0 + j);
                f32x4 h4 = {0.f, 0.f, 0.f, 0.f};
                if (SPLIT) h4 = ld_stream(h + e0 + j);
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    up[4 * k + c] = numerator<SPLIT>(u4[c], h4[c], sc);
                    th[4 * k + c] = t4[c];
                    ss += up[4 * k + c] * up[4 * k + c];
                }
            }
        } else {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int j = lane + kWave * (4 * k + c);
                up[4 * k + c] = 0.f;
                th[4 * k + c] = 0.f;
                if (j < n) {
                    up[4 * k + c] = numerator<SPLIT>(u[e0 + j], SPLIT ? h[e0 + j] : 0.f, sc);
                    th[4 * k + c] = theta[e0 + j];
                    ss += up[4 * k + c] * up[4 * k + c];
                }
            }
        }
    }
    ss = wave_sum(ss);
    const float vb = sc.beta2 * v[b] + sc.one_minus_beta2 * (ss / (float)n);
    if (lane == 0) v[b] = vb;
    const float denom = sqrtf(vb * sc.inv_bc2) + sc.eps;
    const float keep = 1.0f - sc.lr * wd;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        if constexpr (VEC) {
            const int j = (lane + kWave * k) * 4;
            if (j < n) {
                f32x4 t4;
#pragma unroll
                for (int c = 0; c < 4; ++c) t4[c] = keep * th[4 * k + c] - sc.lr * (up[4 * k + c] / denom);
                st_stream(theta + e0 + j, t4);
            }
        } else {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int j = lane + kWave * (4 * k + c);
                if (j < n) theta[e0 + j] = keep * th[4 * k + c] - sc.lr * (up[4 * k + c] / denom);
            }
        }
    }
}

// Blocks longer than kBlkWave: piece p of block b = p / np covers [b blk + (p % np) kBlkWave, +kBlkWave),
// cut at the block's and the segment's end.
__device__ __forceinline__ void piece_range(int64_t p, int np, int64_t blk, int64_t len, int64_t* e0, int* n) {
    const int64_t b = p / np;
    const int64_t s0 = b * blk + (p % np) * (int64_t)kBlkWave;
    int64_t e1 = b * blk + blk < len ? b * blk + blk : len;
    if (s0 + kBlkWave < e1) e1 = s0 + kBlkWave;
    *e0 = s0;
    *n = (int)(e1 - s0);
}

template <bool SPLIT, bool VEC>
__global__ __launch_bounds__(kUpdThreads) void blocks_piece_stats_kernel(const float* __restrict__ u,
                                                                         const float* __restrict__ h, int64_t len,
                                                                         int64_t blk, int64_t npieces, int np,
                                                                         float* __restrict__ part, UpdateScalars sc) {
    const int lane = threadIdx.x % kWave;
    const int64_t p = (int64_t)blockIdx.x * kWavesPerWG + threadIdx.x / kWave;
    if (p >= npieces) return;
    sc = clipped(sc);
    int64_t e0;
    int n;
    piece_range(p, np, blk, len, &e0, &n);
    float ss = 0.f;
    if constexpr (VEC) {
        for (int j = lane * 4; j < n; j += kWave * 4) {
            const f32x4 u4 = ld_stream(u + e0 + j);
            f32x4 h4 = {0.f, 0.f, 0.f, 0.f};
            if (SPLIT) h4 = ld_stream(h + e0 + j);
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const float x = numerator<SPLIT>(u4[c], h4[c], sc);
                ss += x * x;
            }
        }
    } else {
        for (int j = lane; j < n; j += kWave) {
            const float x = numerator<SPLIT>(u[e0 + j], SPLIT ? h[e0 + j] : 0.f, sc);
            ss += x * x;
        }
    }
    ss = wave_sum(ss);
    if (lane == 0) part[p] = ss;
}

// One thread per block: the partial sums in piece order, then the block's second moment.
__global__ __launch_bounds__(kUpdThreads) void blocks_finish_kernel(float* __restrict__ v, const float* __restrict__ part,
                                                                    int64_t nblk, int np, int64_t blk, int64_t len,
                                                                    UpdateScalars sc) {
    const int64_t b = (int64_t)blockIdx.x * kUpdThreads + threadIdx.x;
    if (b >= nblk) return;
    float ss = 0.f;
    for (int q = 0; q < np; ++q) ss += part[b * np + q];
    const int64_t n = b * blk + blk < len ? blk : len - b * blk;
    v[b] = sc.beta2 * v[b] + sc.one_minus_beta2 * (ss / (float)n);
}

template <bool SPLIT, bool VEC>
__global__ __launch_bounds__(kUpdThreads) void blocks_piece_step_kernel(float* __restrict__ theta,
                                                                        const float* __restrict__ v,
                                                                        const float* __restrict__ u,
                                                                        const float* __restrict__ h, int64_t len,
                                                                        int64_t blk, int64_t npieces, int np, float wd,
                                                                        UpdateScalars sc) {
    const int lane = threadIdx.x % kWave;
    const int64_t p = (int64_t)blockIdx.x * kWavesPerWG + threadIdx.x / kWave;
    if (p >= npieces) return;
    sc = clipped(sc);
    int64_t e0;
    int n;
    piece_range(p, np, blk, len, &e0, &n);
    const float denom = sqrtf(v[p / np] * sc.inv_bc2) + sc.eps;
    const float keep = 1.0f - sc.lr * wd;
    if constexpr (VEC) {
        for (int j = lane * 4; j < n; j += kWave * 4) {
            const f32x4 u4 = ld_stream(u + e0 + j);
            f32x4 t4 = ld_stream(theta + e0 + j);
            f32x4 h4 = {0.f, 0.f, 0.f, 0.f};
            if (SPLIT) h4 = ld_stream(h + e0 + j);
#pragma unroll
            for (int c = 0; c < 4; ++c) t4[c] = keep * t4[c] - sc.lr * (numerator<SPLIT>(u4[c], h4[c], sc) / denom);
            st_stream(theta + e0 + j, t4);
        }
    } else {
        for (int j = lane; j < n; j += kWave) {
            const float x = numerator<SPLIT>(u[e0 + j], SPLIT ? h[e0 + j] : 0.f, sc);
            theta[e0 + j] = keep * theta[e0 + j] - sc.lr * (x / denom);
        }
    }
}

constexpr int kClipGroups = 2048;  // workgroups of the norm pass (fixed: the sum order is fixed)
constexpr int kClipUnroll = 4;     // 16-byte groups per thread in flight

// Per-workgroup fp64 partial sums: SQUARE, the sum of squares of the numerator of (u, h) over n
// elements (16-byte groups when aligned); otherwise the plain sum of n values of u (the row sums of
// squares kept by the factored statistics kernel).
template <bool SPLIT, bool SQUARE>
__global__ __launch_bounds__(kUpdThreads) void clip_partial_kernel(const float* __restrict__ u,
                                                                   const float* __restrict__ h, int64_t n,
                                                                   bool vec4, UpdateScalars sc,
                                                                   double* __restrict__ part) {
    __shared__ double sh[kUpdThreads / kWave];
    const int t = threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * kUpdThreads;
    double acc = 0.0;
    int64_t done = 0;
    if (vec4) {
        const int64_t nvec = n / 4;
        int64_t q = (int64_t)blockIdx.x * kUpdThreads + t;
        // kClipUnroll groups per thread in flight, then the remainder one group at a time
        for (; q + (kClipUnroll - 1) * stride < nvec; q += kClipUnroll * stride) {
            f32x4 u4[kClipUnroll], h4[kClipUnroll];
#pragma unroll
            for (int k = 0; k < kClipUnroll; ++k) {
                u4[k] = ld_stream(u + (q + k * stride) * 4);
                h4[k] = SPLIT ? ld_stream(h + (q + k * stride) * 4) : f32x4{0.f, 0.f, 0.f, 0.f};
            }
#pragma unroll
            for (int k = 0; k < kClipUnroll; ++k)
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const double x = SQUARE ? (double)numerator<SPLIT>(u4[k][c], h4[k][c], sc) : (double)u4[k][c];
                    acc += SQUARE ? x * x : x;
                }
        }
        for (; q < nvec; q += stride) {
            const f32x4 u4 = ld_stream(u + q * 4);
            f32x4 h4 = {0.f, 0.f, 0.f, 0.f};
            if (SPLIT) h4 = ld_stream(h + q * 4);
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const double x = SQUARE ? (double)numerator<SPLIT>(u4[c], h4[c], sc) : (double)u4[c];
                acc += SQUARE ? x * x : x;
            }
        }
        done = nvec * 4;
    }
    for (int64_t e = done + (int64_t)blockIdx.x * kUpdThreads + t; e < n; e += stride) {
        const double x = SQUARE ? (double)numerator<SPLIT>(u[e], SPLIT ? h[e] : 0.f, sc) : (double)u[e];
        acc += SQUARE ? x * x : x;
    }
    acc = wave_sum(acc);
    if (t % kWave == 0) sh[t / kWave] = acc;
    __syncthreads();
    if (t == 0) part[blockIdx.x] = ((sh[0] + sh[1]) + sh[2]) + sh[3];
}

// The same partial sums of squares of the numerator for bf16 storage (eight elements per 16 bytes).
template <bool SPLIT>
__global__ __launch_bounds__(kUpdThreads) void clip_partial_bf16_kernel(const uint16_t* __restrict__ u,
                                                                        const uint16_t* __restrict__ h, int64_t n,
                                                                        bool vec8, UpdateScalars sc,
                                                                        double* __restrict__ part) {
    __shared__ double sh[kUpdThreads / kWave];
    const int t = threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * kUpdThreads;
    double acc = 0.0;
    int64_t done = 0;
    if (vec8) {
        const int64_t nvec = n / 8;
        for (int64_t q = (int64_t)blockIdx.x * kUpdThreads + t; q < nvec; q += stride) {
            const u32x4_t u8 = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(u + q * 8));
            u32x4_t h8 = {0u, 0u, 0u, 0u};
            if (SPLIT) h8 = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(h + q * 8));
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                const float uc = c & 1 ? bf16_hi(u8[c / 2]) : bf16_lo(u8[c / 2]);
                const float hc = c & 1 ? bf16_hi(h8[c / 2]) : bf16_lo(h8[c / 2]);
                const double x = (double)numerator<SPLIT>(uc, hc, sc);
                acc += x * x;
            }
        }
        done = nvec * 8;
    }
    for (int64_t e = done + (int64_t)blockIdx.x * kUpdThreads + t; e < n; e += stride) {
        const double x = (double)numerator<SPLIT>(bf16_to_f32(u[e]), SPLIT ? bf16_to_f32(h[e]) : 0.f, sc);
        acc += x * x;
    }
    acc = wave_sum(acc);
    if (t % kWave == 0) sh[t / kWave] = acc;
    __syncthreads();
    if (t == 0) part[blockIdx.x] = ((sh[0] + sh[1]) + sh[2]) + sh[3];
}

// One workgroup: the total of the partial sums (fixed order), ||u'|| = sqrt(total), and the factor
// c = min(1, clip_norm / (||u'|| + 1e-6)) written to clip[0] (and, if requested, norm and factor to
// clip_stats).
__global__ __launch_bounds__(kUpdThreads) void clip_finish_kernel(const double* __restrict__ part, int nparts,
                                                                  float* __restrict__ clip, UpdateScalars sc) {
    __shared__ double sh[kUpdThreads];
    const int t = threadIdx.x;
    double a = 0.0;
    for (int k = t; k < nparts; k += kUpdThreads) a += part[k];
    sh[t] = a;
    __syncthreads();
    for (int o = kUpdThreads / 2; o > 0; o >>= 1) {
        if (t < o) sh[t] += sh[t + o];
        __syncthreads();
    }
    if (t == 0) {
        const double norm = sqrt(sh[0]);
        const double c = (double)sc.clip_norm / (norm + 1e-6);
        const float cf = c < 1.0 ? (float)c : 1.0f;
        clip[0] = cf;
        if (sc.clip_stats) {
            sc.clip_stats[0] = (float)norm;
            sc.clip_stats[1] = cf;
        }
    }
}

// Workspace of the clipping pass: fp64 partials, then the factor word.
struct ClipLayout {
    size_t part_off, clip_off, total;
};
ClipLayout clip_layout(size_t base) {
    ClipLayout L;
    L.part_off = align256(base);
    L.clip_off = align256(L.part_off + (size_t)kClipGroups * sizeof(double));
    L.total = align256(L.clip_off + 16);
    return L;
}

// Norm pass and factor: SQUARE over the numerator (dense), or the plain sum of the row statistics.
template <bool SPLIT, bool SQUARE>
hipError_t run_clip(const float* x, const float* h, int64_t n, bool vec4, UpdateScalars& sc, void* ws,
                    const ClipLayout& L, hipStream_t st) {
    double* part = reinterpret_cast<double*>(static_cast<char*>(ws) + L.part_off);
    float* clip = reinterpret_cast<float*>(static_cast<char*>(ws) + L.clip_off);
    hipLaunchKernelGGL((clip_partial_kernel<SPLIT, SQUARE>), dim3(kClipGroups), dim3(kUpdThreads), 0, st, x, h, n, vec4,
                       sc, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(clip_finish_kernel, dim3(1), dim3(kUpdThreads), 0, st, part, kClipGroups, clip, sc);
    sc.clip = clip;
    return hipGetLastError();
}

struct FacLayout {
    int64_t nrows, nblocks, groups_per_block, ngroups;
    size_t kpart_off, rsum_off, rho_off;
    ClipLayout clip;
    size_t total;
};

FacLayout fac_layout(int64_t P, int64_t br, int64_t bc, bool clip) {
    FacLayout L;
    L.nrows = (P + bc - 1) / bc;
    L.nblocks = (L.nrows + br - 1) / br;
    L.groups_per_block = (br + kFacRowsPerWG - 1) / kFacRowsPerWG;
    L.ngroups = L.nblocks * L.groups_per_block;
    L.kpart_off = 0;
    L.rsum_off = align256((size_t)L.ngroups * (size_t)bc * sizeof(float));
    L.rho_off = align256(L.rsum_off + (size_t)L.nblocks * sizeof(float));
    size_t end = L.rho_off;
    if (clip) {
        L.clip = clip_layout(L.rho_off + (size_t)L.nrows * sizeof(float));
        end = L.clip.total;
    }
    L.total = align256(end);
    return L;
}

template <bool SPLIT, int KC>
hipError_t run_factored(float* theta, float* Rr, float* Cc, const float* u, const float* h, int64_t P, int64_t br,
                        int bc, const SegTable& segs, UpdateScalars sc, void* ws, hipStream_t st) {
    const bool clip = sc.clip_norm > 0.f;
    const FacLayout L = fac_layout(P, br, bc, clip);
    float* kpart = reinterpret_cast<float*>(static_cast<char*>(ws) + L.kpart_off);
    float* rsum = reinterpret_cast<float*>(static_cast<char*>(ws) + L.rsum_off);
    float* rho = clip ? reinterpret_cast<float*>(static_cast<char*>(ws) + L.rho_off) : nullptr;
    // statistics workgroups of the last block beyond its rows simply see an empty row range
    hipLaunchKernelGGL((factored_stats_kernel<SPLIT, KC>), dim3((unsigned)L.ngroups), dim3(kUpdThreads), 0, st, u, h, P,
                       L.nrows, br, bc, (int)L.groups_per_block, Rr, kpart, rho, sc);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (clip && (e = run_clip<false, false>(rho, nullptr, L.nrows, false, sc, ws, L.clip, st)) != hipSuccess) return e;
    hipLaunchKernelGGL(factored_finish_kernel, dim3((unsigned)L.nblocks), dim3(kUpdThreads), 0, st, kpart,
                       (int)L.groups_per_block, L.nrows, br, bc, Rr, Cc, rsum, rho, sc);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const unsigned nupd = (unsigned)((L.nrows + kFacUpdRows - 1) / kFacUpdRows);
    hipLaunchKernelGGL((factored_update_kernel<SPLIT, KC>), dim3(nupd), dim3(kUpdThreads), 0, st, theta, u, h, P,
                       L.nrows, br, bc, Rr, Cc, rsum, segs, sc);
    return hipGetLastError();
}

template <bool SPLIT, int NV>
hipError_t run_factored_rows(float* theta, float* Rr, float* Cc, const float* u, const float* h, int64_t P, int64_t br,
                             const SegTable& segs, UpdateScalars sc, void* ws, hipStream_t st) {
    constexpr int BC = NV * 256;
    const bool clip = sc.clip_norm > 0.f;
    const FacLayout L = fac_layout(P, br, BC, clip);
    float* kpart = reinterpret_cast<float*>(static_cast<char*>(ws) + L.kpart_off);
    float* rsum = reinterpret_cast<float*>(static_cast<char*>(ws) + L.rsum_off);
    float* rho = clip ? reinterpret_cast<float*>(static_cast<char*>(ws) + L.rho_off) : nullptr;
    hipLaunchKernelGGL((factored_stats_rows_kernel<SPLIT, NV>), dim3((unsigned)L.ngroups), dim3(kUpdThreads), 0, st, u, h,
                       P, L.nrows, br, (int)L.groups_per_block, Rr, kpart, rho, sc);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (clip && (e = run_clip<false, false>(rho, nullptr, L.nrows, false, sc, ws, L.clip, st)) != hipSuccess) return e;
    const int nchunks = (BC + 1023) / 1024;
    hipLaunchKernelGGL(factored_finish_cols_kernel, dim3((unsigned)(L.nblocks * nchunks)), dim3(kUpdThreads), 0, st,
                       kpart, (int)L.groups_per_block, L.nrows, br, BC, nchunks, Rr, Cc, rsum, rho, sc);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((factored_update_rows_kernel<SPLIT, NV>), dim3((unsigned)L.nrows), dim3(kUpdThreads), 0, st, theta,
                       u, h, P, br, Rr, Cc, rsum, segs, sc);
    return hipGetLastError();
}

template <bool SPLIT>
hipError_t dispatch_factored(float* theta, float* Rr, float* Cc, const float* u, const float* h, int64_t P, int64_t br,
                             int bc, const SegTable& segs, const UpdateScalars& sc, void* ws, hipStream_t st) {
    // whole-row kernels for block_cols of 1024, 2048 or 4096; the column-strip kernels otherwise
    if (bc == 4096) return run_factored_rows<SPLIT, 16>(theta, Rr, Cc, u, h, P, br, segs, sc, ws, st);
    if (bc == 2048) return run_factored_rows<SPLIT, 8>(theta, Rr, Cc, u, h, P, br, segs, sc, ws, st);
    if (bc == 1024) return run_factored_rows<SPLIT, 4>(theta, Rr, Cc, u, h, P, br, segs, sc, ws, st);
    const int kc = (bc + 1023) / 1024;
    if (kc <= 1) return run_factored<SPLIT, 1>(theta, Rr, Cc, u, h, P, br, bc, segs, sc, ws, st);
    if (kc <= 2) return run_factored<SPLIT, 2>(theta, Rr, Cc, u, h, P, br, bc, segs, sc, ws, st);
    if (kc <= 4) return run_factored<SPLIT, 4>(theta, Rr, Cc, u, h, P, br, bc, segs, sc, ws, st);
    if (kc <= 8) return run_factored<SPLIT, 8>(theta, Rr, Cc, u, h, P, br, bc, segs, sc, ws, st);
    return run_factored<SPLIT, 16>(theta, Rr, Cc, u, h, P, br, bc, segs, sc, ws, st);
}

}  // namespace

size_t update_workspace_bytes(int64_t P, const bom_update_cfg* cfg) {
    if (!cfg || P < 1) return 0;
    const bool clip = cfg->clip_norm > 0.f;
    if (cfg->v_layout == BOM_V_BLOCKS) return clip ? clip_layout(blocks_part_bytes(P)).total : blocks_part_bytes(P);
    if (cfg->v_layout != BOM_V_FACTORED) return clip ? clip_layout(0).total : 0;
    if (cfg->block_rows < 1 || cfg->block_cols < 1) return 0;
    return fac_layout(P, cfg->block_rows, cfg->block_cols, clip).total;
}

namespace {
bool aligned16(const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; }

// Elements before the first 16-byte boundary of arrays that share their offset inside a 16-byte group
// (esz-byte elements, esz-aligned pointers), or -1 when the offsets differ (or a pointer is not esz-aligned).
int64_t common_head(std::initializer_list<const void*> ptrs, int esz) {
    int64_t off = -1;
    for (const void* p : ptrs) {
        if (p == nullptr) continue;
        const int64_t o = (int64_t)(reinterpret_cast<uintptr_t>(p) % 16);
        if (o % esz != 0 || (off >= 0 && o != off)) return -1;
        off = o;
    }
    return off <= 0 ? 0 : (16 - off) / esz;
}

// The dense kernels over P elements (the clipping factor, if any, already in sc.clip): one launch, with a
// scalar head up to the arrays' common 16-byte boundary and a scalar tail; arrays with different offsets
// inside a 16-byte group take the scalar kernel.
hipError_t dense_range(float* theta, float* v, const float* u, const float* h, int64_t P, const SegTable& segs,
                       const UpdateScalars& sc, hipStream_t st) {
    int64_t head = common_head({theta, v, u, h}, 4);
    if (head >= 0) {
        head = std::min(head, P);
        const int64_t nvec = (P - head) / 4;
        const int64_t extra = P - 4 * nvec;   // head + tail elements, one thread each
        const int64_t grid = (nvec + extra + kUpdThreads - 1) / kUpdThreads;
        if (h)
            hipLaunchKernelGGL(update_dense_vec4_kernel<true>, dim3((unsigned)grid), dim3(kUpdThreads), 0, st, theta, v, u,
                               h, head, nvec, P, segs, sc);
        else
            hipLaunchKernelGGL(update_dense_vec4_kernel<false>, dim3((unsigned)grid), dim3(kUpdThreads), 0, st, theta, v,
                               u, h, head, nvec, P, segs, sc);
        return hipGetLastError();
    }
    int64_t grid = (P + kUpdThreads - 1) / kUpdThreads;
    if (grid > 8192) grid = 8192;
    if (h)
        hipLaunchKernelGGL(update_dense_scalar_kernel<true>, dim3((unsigned)grid), dim3(kUpdThreads), 0, st, theta, v, u,
                           h, (int64_t)0, P, segs, sc);
    else
        hipLaunchKernelGGL(update_dense_scalar_kernel<false>, dim3((unsigned)grid), dim3(kUpdThreads), 0, st, theta, v, u,
                           h, (int64_t)0, P, segs, sc);
    return hipGetLastError();
}

// Global-norm clipping pass over the whole numerator: sets sc.clip (no-op without clipping).
hipError_t clip_pass(const float* u, const float* h, int64_t P, UpdateScalars& sc, void* ws, hipStream_t st) {
    if (!(sc.clip_norm > 0.f)) return hipSuccess;
    const bool aligned = aligned16(u) && (h == nullptr || aligned16(h));
    return h ? run_clip<true, true>(u, h, P, aligned, sc, ws, clip_layout(0), st)
             : run_clip<false, true>(u, h, P, aligned, sc, ws, clip_layout(0), st);
}

template <bool SPLIT, int NV>
hipError_t blocks_wave(float* theta, float* v, const float* u, const float* h, int64_t len, int64_t blk, bool vec,
                       float wd, const UpdateScalars& sc, hipStream_t st) {
    const int64_t nblk = (len + blk - 1) / blk;
    const dim3 grid((unsigned)((nblk + kWavesPerWG - 1) / kWavesPerWG));
    if (vec)
        hipLaunchKernelGGL((blocks_wave_kernel<SPLIT, NV, true>), grid, dim3(kUpdThreads), 0, st, theta, v, u, h, len, blk,
                           nblk, wd, sc);
    else
        hipLaunchKernelGGL((blocks_wave_kernel<SPLIT, NV, false>), grid, dim3(kUpdThreads), 0, st, theta, v, u, h, len,
                           blk, nblk, wd, sc);
    return hipGetLastError();
}

template <bool SPLIT>
hipError_t blocks_pieces(float* theta, float* v, const float* u, const float* h, int64_t len, int64_t blk, bool vec,
                         float wd, const UpdateScalars& sc, float* part, hipStream_t st) {
    const int64_t nblk = (len + blk - 1) / blk;
    const int64_t eff = blk < len ? blk : len;   // a block longer than the segment is the segment
    const int np = (int)((eff + kBlkWave - 1) / kBlkWave);
    const int64_t npieces = nblk * np;
    const dim3 grid((unsigned)((npieces + kWavesPerWG - 1) / kWavesPerWG));
    if (vec)
        hipLaunchKernelGGL((blocks_piece_stats_kernel<SPLIT, true>), grid, dim3(kUpdThreads), 0, st, u, h, len, blk,
                           npieces, np, part, sc);
    else
        hipLaunchKernelGGL((blocks_piece_stats_kernel<SPLIT, false>), grid, dim3(kUpdThreads), 0, st, u, h, len, blk,
                           npieces, np, part, sc);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(blocks_finish_kernel, dim3((unsigned)((nblk + kUpdThreads - 1) / kUpdThreads)), dim3(kUpdThreads),
                       0, st, v, part, nblk, np, blk, len, sc);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (vec)
        hipLaunchKernelGGL((blocks_piece_step_kernel<SPLIT, true>), grid, dim3(kUpdThreads), 0, st, theta, v, u, h, len,
                           blk, npieces, np, wd, sc);
    else
        hipLaunchKernelGGL((blocks_piece_step_kernel<SPLIT, false>), grid, dim3(kUpdThreads), 0, st, theta, v, u, h, len,
                           blk, npieces, np, wd, sc);
    return hipGetLastError();
}

template <bool SPLIT>
hipError_t blocks_segment(float* theta, float* v, const float* u, const float* h, int64_t len, int64_t blk, float wd,
                          const UpdateScalars& sc, float* part, hipStream_t st) {
    if (blk == 1) {
        SegTable one{};
        one.n = 0;
        one.wd_default = wd;
        return dense_range(theta, v, u, h, len, one, sc, st);
    }
    const bool vec = aligned16(theta) && aligned16(u) && (h == nullptr || aligned16(h)) && blk % 4 == 0 && len % 4 == 0;
    const int64_t eff = blk < len ? blk : len;
    if (eff <= 256) return blocks_wave<SPLIT, 1>(theta, v, u, h, len, blk, vec, wd, sc, st);
    if (eff <= 1024) return blocks_wave<SPLIT, 4>(theta, v, u, h, len, blk, vec, wd, sc, st);
    if (eff <= kBlkWave) return blocks_wave<SPLIT, 16>(theta, v, u, h, len, blk, vec, wd, sc, st);
    return blocks_pieces<SPLIT>(theta, v, u, h, len, blk, vec, wd, sc, part, st);
}

}  // namespace

hipError_t launch_update_dense(float* theta, float* v, const float* u, const float* h, int64_t P, const SegTable& segs,
                               UpdateScalars sc, void* ws, hipStream_t st) {
    const hipError_t e = clip_pass(u, h, P, sc, ws, st);
    if (e != hipSuccess) return e;
    return dense_range(theta, v, u, h, P, segs, sc, st);
}

int64_t blocks_count(const BlockSegs& b) {
    int64_t n = 0;
    for (int k = 0; k < b.n; ++k) n += (b.len[k] + b.blk[k] - 1) / b.blk[k];
    return n;
}

// Workspace: the partial sums of long blocks (at most 3 per 4096 elements of a segment plus one per
// segment: bounded by P / 1024 + 64 floats), then the clipping pass.
hipError_t launch_update_blocks(float* theta, float* v, const float* u, const float* h, int64_t P, const BlockSegs& bs,
                                UpdateScalars sc, void* ws, hipStream_t st) {
    const size_t pb = blocks_part_bytes(P);
    if (sc.clip_norm > 0.f) {
        const bool aligned = aligned16(u) && (h == nullptr || aligned16(h));
        const hipError_t e = h ? run_clip<true, true>(u, h, P, aligned, sc, ws, clip_layout(pb), st)
                               : run_clip<false, true>(u, h, P, aligned, sc, ws, clip_layout(pb), st);
        if (e != hipSuccess) return e;
    }
    float* part = static_cast<float*>(ws);
    int64_t vb = 0, pused = 0;
    for (int k = 0; k < bs.n; ++k) {
        const int64_t o = bs.begin[k], len = bs.len[k], blk = bs.blk[k];
        const hipError_t e = h ? blocks_segment<true>(theta + o, v + vb, u + o, h + o, len, blk, bs.wd[k], sc, part + pused, st)
                               : blocks_segment<false>(theta + o, v + vb, u + o, nullptr, len, blk, bs.wd[k], sc,
                                                       part + pused, st);
        if (e != hipSuccess) return e;
        const int64_t nblk = (len + blk - 1) / blk;
        const int64_t eff = blk < len ? blk : len;
        if (eff > kBlkWave) pused += nblk * ((eff + kBlkWave - 1) / kBlkWave);
        vb += nblk;
    }
    return hipSuccess;
}

hipError_t launch_update_dense_bf16(uint16_t* theta, uint16_t* v, const uint16_t* u, const uint16_t* h, int64_t P,
                                    const SegTable& segs, UpdateScalars sc, void* ws, hipStream_t st) {
    auto al = [](const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; };
    const bool aligned = al(theta) && al(v) && al(u) && (h == nullptr || al(h));
    if (sc.clip_norm > 0.f) {
        const ClipLayout L = clip_layout(0);
        double* part = reinterpret_cast<double*>(static_cast<char*>(ws) + L.part_off);
        float* clip = reinterpret_cast<float*>(static_cast<char*>(ws) + L.clip_off);
        if (h)
            hipLaunchKernelGGL(clip_partial_bf16_kernel<true>, dim3(kClipGroups), dim3(kUpdThreads), 0, st, u, h, P,
                               aligned, sc, part);
        else
            hipLaunchKernelGGL(clip_partial_bf16_kernel<false>, dim3(kClipGroups), dim3(kUpdThreads), 0, st, u, h, P,
                               aligned, sc, part);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(clip_finish_kernel, dim3(1), dim3(kUpdThreads), 0, st, part, kClipGroups, clip, sc);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        sc.clip = clip;
    }
    int64_t head = common_head({theta, v, u, h}, 2);
    if (head >= 0) {
        head = std::min(head, P);
        const int64_t nvec = (P - head) / 8;
        const int64_t extra = P - 8 * nvec;   // head + tail elements, one thread each
        const int64_t grid = (nvec + extra + kUpdThreads - 1) / kUpdThreads;
        if (h)
            hipLaunchKernelGGL(update_dense_bf16x8_kernel<true>, dim3((unsigned)grid), dim3(kUpdThreads), 0, st, theta, v,
                               u, h, head, nvec, P, segs, sc);
        else
            hipLaunchKernelGGL(update_dense_bf16x8_kernel<false>, dim3((unsigned)grid), dim3(kUpdThreads), 0, st, theta, v,
                               u, h, head, nvec, P, segs, sc);
        return hipGetLastError();
    }
    int64_t grid = (P + kUpdThreads - 1) / kUpdThreads;
    if (grid > 8192) grid = 8192;
    if (h)
        hipLaunchKernelGGL(update_dense_bf16_scalar_kernel<true>, dim3((unsigned)grid), dim3(kUpdThreads), 0, st, theta, v,
                           u, h, (int64_t)0, P, segs, sc);
    else
        hipLaunchKernelGGL(update_dense_bf16_scalar_kernel<false>, dim3((unsigned)grid), dim3(kUpdThreads), 0, st, theta, v,
                           u, h, (int64_t)0, P, segs, sc);
    return hipGetLastError();
}

hipError_t launch_update_factored(float* theta, float* Rr, float* Cc, const float* u, const float* h, int64_t P,
                                  int64_t block_rows, int64_t block_cols, const SegTable& segs,
                                  const UpdateScalars& sc, void* ws, hipStream_t st) {
    if (h) return dispatch_factored<true>(theta, Rr, Cc, u, h, P, block_rows, (int)block_cols, segs, sc, ws, st);
    return dispatch_factored<false>(theta, Rr, Cc, u, h, P, block_rows, (int)block_cols, segs, sc, ws, st);
}

hipError_t launch_adamw_dense(float* theta, float* m, float* v, const float* g, int64_t P, const SegTable& segs,
                              const UpdateScalars& sc, hipStream_t st) {
    int64_t head = common_head({theta, m, v, g}, 4);
    if (head >= 0) {
        head = std::min(head, P);
        const int64_t nvec = (P - head) / 4;
        const int64_t grid = (nvec + (P - 4 * nvec) + kUpdThreads - 1) / kUpdThreads;
        hipLaunchKernelGGL(adamw_dense_vec4_kernel, dim3((unsigned)grid), dim3(kUpdThreads), 0, st, theta, m, v, g, head,
                           nvec, P, segs, sc);
        return hipGetLastError();
    }
    const int64_t grid = std::min<int64_t>((P + kUpdThreads - 1) / kUpdThreads, 8192);
    hipLaunchKernelGGL(adamw_dense_scalar_kernel, dim3((unsigned)grid), dim3(kUpdThreads), 0, st, theta, m, v, g, P, segs,
                       sc);
    return hipGetLastError();
}

namespace {
template <int NV>
hipError_t run_adamw_factored_rows(float* theta, float* m, float* Rr, float* Cc, const float* g, int64_t P, int64_t br,
                                   const SegTable& segs, const UpdateScalars& sc, void* ws, hipStream_t st) {
    constexpr int BC = NV * 256;
    const FacLayout L = fac_layout(P, br, BC, false);
    float* kpart = reinterpret_cast<float*>(static_cast<char*>(ws) + L.kpart_off);
    float* rsum = reinterpret_cast<float*>(static_cast<char*>(ws) + L.rsum_off);
    // the second moment's statistics are those of the factored BOM update with numerator g
    hipLaunchKernelGGL((factored_stats_rows_kernel<false, NV>), dim3((unsigned)L.ngroups), dim3(kUpdThreads), 0, st, g,
                       nullptr, P, L.nrows, br, (int)L.groups_per_block, Rr, kpart, nullptr, sc);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int nchunks = (BC + 1023) / 1024;
    hipLaunchKernelGGL(factored_finish_cols_kernel, dim3((unsigned)(L.nblocks * nchunks)), dim3(kUpdThreads), 0, st,
                       kpart, (int)L.groups_per_block, L.nrows, br, BC, nchunks, Rr, Cc, rsum, nullptr, sc);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL((factored_adamw_rows_kernel<NV>), dim3((unsigned)L.nrows), dim3(kUpdThreads), 0, st, theta, m, g,
                       P, br, Rr, Cc, rsum, segs, sc);
    return hipGetLastError();
}
}  // namespace

hipError_t launch_adamw_factored(float* theta, float* m, float* Rr, float* Cc, const float* g, int64_t P,
                                 int64_t block_rows, int64_t block_cols, const SegTable& segs, const UpdateScalars& sc,
                                 void* ws, hipStream_t st) {
    if (block_cols == 4096) return run_adamw_factored_rows<16>(theta, m, Rr, Cc, g, P, block_rows, segs, sc, ws, st);
    if (block_cols == 2048) return run_adamw_factored_rows<8>(theta, m, Rr, Cc, g, P, block_rows, segs, sc, ws, st);
    if (block_cols == 1024) return run_adamw_factored_rows<4>(theta, m, Rr, Cc, g, P, block_rows, segs, sc, ws, st);
    return hipErrorInvalidValue;
}

}  // namespace bom
