// bom_head_vjp kernels: the output-head part of the one backward pass through the mixed
// objective (Eq. (3)); its gradient (Eq. (4)) for the linear head z_i = W^T h_i (+ b) is
//   G_ij = [i in I] ((1 - lambda) R_ij + lambda q_hat_j) / N_t      (gradient w.r.t. the logits)
//   dW = H^T G,  dH = G W^T,  db = 1^T G = (1 - lambda) s + lambda q_hat  (bias Jacobian = I).
// G is never stored. The large products (and the fused launch for small ones) use its rank-1 split
//   dW = alpha H^T R + hsum cq^T,  dH = alpha R W^T + mask u^T,
//   alpha = (1 - lambda) / N_t,  cq_j = lambda q_hat_j / N_t,  hsum = sum over rows in I of H,  u = W cq,
// multiplying R as stored; the 128-tile split-K kernels instead form G = fma(alpha, R, mask_i * cq_j)
// while staging R into LDS and round it to bf16 for the MFMA.
//
// bf16 path: v_mfma_f32_32x32x16_bf16. Large products: 256 x 256 output tiles, eight waves (two per
// SIMD) each owning 128 x 64, k tiles of 64 in two LDS stages (lds256w_kernel). Small products: one fused launch of
// 64 x 64 tiles of both products (vjp_fused_small_kernel), or 128 x 128 split-K tiles with a
// fixed-order reduction. dW = H^T G has both operands k-outer in memory (transposing LDS reads or a
// transpose while staging); dH = G W^T has both operands k-contiguous. fp32 path (and unaligned
// bf16): a SIMT tiled GEMM.
#include <algorithm>
#include <array>
#include <map>
#include <mutex>
#include <queue>
#include <vector>
#include <cstdio>
#include <cstdlib>
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace bom {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;

struct Fold {
    const float* cq;     // [V] lambda * q_hat / N_t
    const float* vmask;  // [N] 1 for rows in I, else 0
    const float* scal;   // [0] alpha = (1 - lambda) / N_t; [1] s_out; [2], [3] bf16 pairs (r_coef, 0), (0, r_coef)
    const float* cqp;    // [V] history term of the rescaled fold G = s_out * (r_coef * R + cqp)
    const float* zc;     // logits input: [N] lse_i log2 e for rows in I, +inf otherwise; null: R is stored
    const int32_t* labels;
};

struct VjpWs {
    size_t cq_off, cqp_off, vmask_off, scal_off, zc_off, hpart_off, hsum_off, u_off, upart_off, part_off, total;
};

// Rank-1 vector u = W q_hat is summed over column chunks (one wave per row of W and chunk at a time, four
// 16-byte loads of W in flight per lane); the chunk sums are added in chunk order by the prep kernel. Rows
// are cut into as many chunks as bring the work to about 4096 units (a short row count, as at d = 768, needs
// several per row; d = 4096 rows need none), each a multiple of the 2048 columns a wave covers per
// iteration, and kUWaves waves take the units in turn: 1024 or 4096 waves measured slower at the three LM
// shapes (at d = 4096, 359 and 300 against 264 us).
constexpr int kUWaves = 2048;
inline int u_chunk_cols(int64_t d, int64_t V) {
    const int64_t c = std::max<int64_t>(1, std::min<int64_t>((4096 + d - 1) / d, (V + 2047) / 2048));
    return (int)(((V + c - 1) / c + 2047) / 2048 * 2048);
}
inline int u_chunks(int64_t d, int64_t V) {   // every chunk starts inside the row
    const int64_t cw = u_chunk_cols(d, V);
    return (int)((V + cw - 1) / cw);
}

// ---- residual rows from the logits ----------------------------------------------------------------
// With the logits Z as input, the products take R = softmax(Z) - onehot(y) chunk by chunk as the operand
// copies pass through registers: r = exp2(z log2 e - c_i) with c_i = lse_i log2 e (c_i = +inf for rows
// outside I, so their r is 0), minus 1 at column y_i, rounded once to the operand type -- the operations
// bom_residual uses when it writes R, so R is the same whether it is stored or formed here.
__device__ __forceinline__ float r_from_z(float z, float c, bool at_label) {
    float p = exp2_fast(fmaf(z, kLog2e, -c));
    if (at_label) p -= 1.0f;
    return p;
}
// Eight bf16 logits of one row (columns j0 .. j0 + 7, lab_off = y_i - j0) to eight bf16 residuals; ok = false
// gives zeros (a chunk outside the operand).
__device__ __forceinline__ u32x4_t z_chunk_to_r(u32x4_t z, float c, int lab_off, bool ok) {
    u32x4_t r;
#pragma unroll
    for (int p = 0; p < 4; ++p)
        r[p] = pack_bf16x2(r_from_z(bf16_lo(z[p]), c, lab_off == 2 * p), r_from_z(bf16_hi(z[p]), c, lab_off == 2 * p + 1));
    const uint32_t mk = lane_mask(ok);
    return u32x4_t{r[0] & mk, r[1] & mk, r[2] & mk, r[3] & mk};
}
// c_i of row i from lse and the label (the fused kernel forms it itself)
__device__ __forceinline__ float z_row_c(const float* row_lse, const int32_t* labels, int i, int V, int32_t ig) {
    bool bad = false;
    return label_valid(labels[i], V, ig, &bad) ? row_lse[i] * kLog2e : INFINITY;
}

// ---- prep -------------------------------------------------------------------------------------
// G = alpha R + mask * cq  (alpha = (1-lambda)/N_t, cq = lambda q_hat / N_t) is also written
// G = s_out (r_coef R + mask * cqp): for lambda < 1, s_out = alpha, r_coef = 1, cqp = lambda/(1-lambda) q_hat;
// for lambda = 1, s_out = 1/N_t, r_coef = 0, cqp = q_hat. The large-tile kernels fold cqp with one
// bf16 dot product per element and apply s_out to the fp32 accumulators.
__global__ __launch_bounds__(256) void vjp_prep_kernel(const float* __restrict__ q_hat, const float* __restrict__ s,
                                                       const int32_t* __restrict__ n_valid, float lambda, int V, int N,
                                                       const int32_t* __restrict__ labels, int32_t ignore_index,
                                                       float* __restrict__ cq, float* __restrict__ cqp,
                                                       float* __restrict__ vmask, float* __restrict__ scal,
                                                       float* __restrict__ db, const float* __restrict__ hpart, int nrb,
                                                       int d, float* __restrict__ hsum, const float* __restrict__ row_lse,
                                                       float* __restrict__ zc, const float* __restrict__ upart, int uch,
                                                       float* __restrict__ u) {
    const int idx = blockIdx.x * 256 + threadIdx.x;
    const int nt = *n_valid;
    if (hpart != nullptr && idx < d) {   // rank-1 form: hsum_m = sum of the row-block partials, in block order
        float a = 0.f;
        int b = 0;
        for (; b + 8 <= nrb; b += 8) {   // eight loads in flight, added in block order
            float h[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) h[k] = hpart[(int64_t)(b + k) * d + idx];
#pragma unroll
            for (int k = 0; k < 8; ++k) a += h[k];
        }
        for (; b < nrb; ++b) a += hpart[(int64_t)b * d + idx];
        hsum[idx] = a;
    }
    if (upart != nullptr && idx < d) {   // u_n = (lambda / N_t) sum of the chunk sums, in chunk order
        float a = 0.f;
        for (int c = 0; c < uch; ++c) a += upart[(int64_t)c * d + idx];
        u[idx] = nt > 0 ? (float)((double)lambda / (double)nt) * a : 0.f;
    }
    const bool hist_only = !(lambda < 1.0f);
    if (idx < V) {
        cq[idx] = nt > 0 ? (float)((double)lambda * (double)q_hat[idx] / (double)nt) : 0.f;
        cqp[idx] = hist_only ? q_hat[idx] : (float)((double)lambda / (1.0 - (double)lambda) * (double)q_hat[idx]);
        if (db) db[idx] = nt > 0 ? (1.0f - lambda) * s[idx] + lambda * q_hat[idx] : 0.f;
    }
    if (idx < N) {
        bool bad = false;
        const bool valid = label_valid(labels[idx], V, ignore_index, &bad);
        vmask[idx] = valid ? 1.f : 0.f;
        if (row_lse != nullptr) zc[idx] = valid ? row_lse[idx] * kLog2e : INFINITY;
    }
    if (idx == 0) {
        scal[0] = nt > 0 ? (float)((1.0 - (double)lambda) / (double)nt) : 0.f;
        scal[1] = nt > 0 ? (hist_only ? (float)(1.0 / (double)nt) : scal[0]) : 0.f;
        const uint32_t one = hist_only ? 0u : 0x3F80u;   // bf16 1.0 (or 0 when R drops out)
        scal[2] = __uint_as_float(one);
        scal[3] = __uint_as_float(one << 16);
    }
}

template <typename T>
__device__ __forceinline__ float ldf(const T* p, int64_t i);
template <>
__device__ __forceinline__ float ldf<float>(const float* p, int64_t i) { return p[i]; }
template <>
__device__ __forceinline__ float ldf<uint16_t>(const uint16_t* p, int64_t i) { return bf16_to_f32(p[i]); }

template <typename T>
__device__ __forceinline__ void stf(T* p, int64_t i, float x);
template <>
__device__ __forceinline__ void stf<float>(float* p, int64_t i, float x) { p[i] = x; }
template <>
__device__ __forceinline__ void stf<uint16_t>(uint16_t* p, int64_t i, float x) { p[i] = f32_to_bf16(x); }

// Element (row, col) of R: as stored, or formed from the logits (rounded to T like a stored R).
template <typename T>
__device__ __forceinline__ float r_elem(const T* RZ, int64_t ld, int row, int col, const Fold& f) {
    const float x = ldf(RZ, (int64_t)row * ld + col);
    if (f.zc == nullptr) return x;
    const float p = r_from_z(x, f.zc[row], col == f.labels[row]);
    if constexpr (std::is_same<T, uint16_t>::value) return bf16_to_f32(f32_to_bf16(p));
    return p;
}

// ---- SIMT fallback: 64 x 64 tiles, 16-deep k, 4 x 4 outputs per thread --------------------------
constexpr int SB = 64, SK = 16;

// dW[m][n] = sum_k H[k][m] G[k][n];  M = d, Nn = V, K = N rows.
template <typename T>
__global__ __launch_bounds__(256) void simt_dW_kernel(const T* __restrict__ H, int64_t ldh, const T* __restrict__ R,
                                                      int64_t ldr, int M, int Nn, int K, int kps, Fold f,
                                                      float* __restrict__ out, int64_t ldo, float beta, int direct) {
    __shared__ float As[SK][SB + 4];
    __shared__ float Bs[SK][SB + 4];
    const int t = threadIdx.x, tx = t % 16, ty = t / 16;
    const int m0 = blockIdx.y * SB, n0 = blockIdx.x * SB;
    const int kb = blockIdx.z * kps, ke = min(K, kb + kps);
    const float alpha = f.scal[0];
    float acc[4][4] = {};
    for (int k0 = kb; k0 < ke; k0 += SK) {
        for (int e = 0; e < 4; ++e) {
            const int idx = e * 256 + t, kk = idx / SB, cc = idx % SB;
            const int k = k0 + kk;
            As[kk][cc] = (k < ke && m0 + cc < M) ? ldf(H, (int64_t)k * ldh + m0 + cc) : 0.f;
            Bs[kk][cc] = (k < ke && n0 + cc < Nn) ? fmaf(alpha, r_elem(R, ldr, k, n0 + cc, f), f.vmask[k] * f.cq[n0 + cc]) : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < SK; ++kk) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
    for (int i = 0; i < 4; ++i)
        for (int j = 0; j < 4; ++j) {
            const int m = m0 + ty * 4 + i, n = n0 + tx * 4 + j;
            if (m >= M || n >= Nn) continue;
            if (direct) {
                float v = acc[i][j];
                if (beta != 0.f) v += beta * out[(int64_t)m * ldo + n];
                out[(int64_t)m * ldo + n] = v;
            } else {
                out[((int64_t)blockIdx.z * M + m) * Nn + n] = acc[i][j];
            }
        }
}

// dH[i][n] = sum_j G[i][j] W[n][j];  M = N rows, Nn = d, K = V.
template <typename T, typename TO>
__global__ __launch_bounds__(256) void simt_dH_kernel(const T* __restrict__ R, int64_t ldr, const T* __restrict__ W,
                                                      int64_t ldw, int M, int Nn, int K, int kps, Fold f,
                                                      TO* __restrict__ out, int64_t ldo, float* __restrict__ part,
                                                      int direct) {
    __shared__ float As[SK][SB + 4];
    __shared__ float Bs[SK][SB + 4];
    const int t = threadIdx.x, tx = t % 16, ty = t / 16;
    const int m0 = blockIdx.y * SB, n0 = blockIdx.x * SB;
    const int kb = blockIdx.z * kps, ke = min(K, kb + kps);
    const float alpha = f.scal[0];
    float acc[4][4] = {};
    for (int k0 = kb; k0 < ke; k0 += SK) {
        for (int e = 0; e < 4; ++e) {
            const int idx = e * 256 + t, rr = idx / SK, kk = idx % SK;
            const int k = k0 + kk;
            As[kk][rr] = (k < ke && m0 + rr < M) ? fmaf(alpha, r_elem(R, ldr, m0 + rr, k, f), f.vmask[m0 + rr] * f.cq[k]) : 0.f;
            Bs[kk][rr] = (k < ke && n0 + rr < Nn) ? ldf(W, (int64_t)(n0 + rr) * ldw + k) : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < SK; ++kk) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
    for (int i = 0; i < 4; ++i)
        for (int j = 0; j < 4; ++j) {
            const int m = m0 + ty * 4 + i, n = n0 + tx * 4 + j;
            if (m >= M || n >= Nn) continue;
            if (direct) stf<TO>(out, (int64_t)m * ldo + n, acc[i][j]);
            else part[((int64_t)blockIdx.z * M + m) * Nn + n] = acc[i][j];
        }
}

// ---- fp32 small heads in one launch -------------------------------------------------------------------
// Both products of a small fp32 head (the tiny classifier) in one grid, each workgroup one 64 x 64 SIMT tile
// of dW (blocks [0, tw)) or of dH (the rest) over the whole k range in chunks of 64, with G folded in as its operand is
// staged: G_ij = [i in I] (alpha R_ij + cq_j), alpha = (1 - lambda) / N_t, cq_j = lambda q_hat_j / N_t,
// formed here from the device words (no prep kernel); R may come from the logits (row_lse given). Block 0
// also writes db = (1 - lambda) s + lambda q_hat.
struct SmallF32Args {
    const float* H; int64_t ldh;
    const float* W; int64_t ldw;
    const float* R; int64_t ldr;
    const float* row_lse;   // logits input: R formed from Z and lse; null: R is stored
    const int32_t* labels; int32_t ig;
    const float* q_hat; const float* s; const int32_t* n_valid; float lambda;
    int N, d, V;
    float* dW; int64_t lddw; float beta;
    float* db;
    void* dH; int64_t lddh; int dh_bf16;
    int tw_n, tw, th_n;
};

__global__ __launch_bounds__(256) void vjp_small_f32_kernel(SmallF32Args a) {
    constexpr int FK = 64;   // k chunk: every load of a chunk (16 per operand per thread) is in flight at once
    __shared__ float As[FK][SB + 4];
    __shared__ float Bs[FK][SB + 4];
    const bool is_dw = (int)blockIdx.x < a.tw;
    const int id = is_dw ? blockIdx.x : blockIdx.x - a.tw;
    const int tn_count = is_dw ? a.tw_n : a.th_n;
    const int m0 = (id / tn_count) * SB, n0 = (id % tn_count) * SB;
    const int M = is_dw ? a.d : a.N, Nn = is_dw ? a.V : a.d, K = is_dw ? a.N : a.V;
    const int t = threadIdx.x, tx = t % 16, ty = t / 16;
    // a tile with at most 16 columns inside the output (the classifier's dW over 10 classes) maps its threads
    // to 64 rows x 4 column groups, so no thread spends its products on columns past the output
    const bool narrow = Nn - n0 <= 16;
    const int nr = t / 4, nc = t % 4;
    const int nt = *a.n_valid;
    const float alpha = nt > 0 ? (float)((1.0 - (double)a.lambda) / (double)nt) : 0.f;
    const double cs = nt > 0 ? (double)a.lambda / (double)nt : 0.0;
    // G element of row i, column j from its loaded words (label y, R or Z value r, the row's lse, q_hat_j)
    const bool zin = a.row_lse != nullptr;
    auto g_from = [&](float r, int y, float lse, float q, int j) {
        bool bad = false;
        if (zin) r = r_from_z(r, lse * kLog2e, j == y);
        return label_valid(y, a.V, a.ig, &bad) ? fmaf(alpha, r, (float)(cs * (double)q)) : 0.f;
    };
    // without the logits input the lse loads read q_hat[0] (a valid word whose value is not used), so that
    // no load of the staging is conditional: all of a chunk's loads are then issued before the first wait
    const float* lse_src = zin ? a.row_lse : a.q_hat;
    const int lse_on = zin ? 1 : 0;
    constexpr int EPT = FK * SB / 256;   // staged elements per thread and operand
    float acc[4][4] = {};
    // a chunk's words are loaded into registers one chunk ahead (issued right after the previous chunk was
    // staged, so they are in flight during its products), from clamped in-range addresses; the product
    // test is outside the unrolled loops, which keeps each chunk's loads together
    float xa[EPT], xr[EPT], xl[EPT], xq[EPT];
    int xy[EPT];
    auto load_chunk = [&](int k0) {
        if (is_dw) {   // A(m, k) = H[k][m], B(k, n) = G[k][n]
#pragma unroll
            for (int e = 0; e < EPT; ++e) {
                const int idx = e * 256 + t, kk = idx / SB, cc = idx % SB;
                const int kc = min(k0 + kk, K - 1), mc = min(m0 + cc, M - 1), nc = min(n0 + cc, Nn - 1);
                xa[e] = a.H[(int64_t)kc * a.ldh + mc];
                xr[e] = a.R[(int64_t)kc * a.ldr + nc];
                xy[e] = a.labels[kc];
                xl[e] = lse_src[kc * lse_on];
                xq[e] = a.q_hat[nc];
            }
        } else {       // A(i, k) = G[i][k], B(k, n) = W[n][k]
#pragma unroll
            for (int e = 0; e < EPT; ++e) {
                const int idx = e * 256 + t, rr = idx / FK, kk = idx % FK;
                const int kc = min(k0 + kk, K - 1), ic = min(m0 + rr, M - 1), nc = min(n0 + rr, Nn - 1);
                xa[e] = a.W[(int64_t)nc * a.ldw + kc];
                xr[e] = a.R[(int64_t)ic * a.ldr + kc];
                xy[e] = a.labels[ic];
                xl[e] = lse_src[ic * lse_on];
                xq[e] = a.q_hat[kc];
            }
        }
    };
    load_chunk(0);
    for (int k0 = 0; k0 < K; k0 += FK) {
        if (is_dw) {
#pragma unroll
            for (int e = 0; e < EPT; ++e) {
                const int idx = e * 256 + t, kk = idx / SB, cc = idx % SB, k = k0 + kk;
                As[kk][cc] = (k < K && m0 + cc < M) ? xa[e] : 0.f;
                Bs[kk][cc] = (k < K && n0 + cc < Nn) ? g_from(xr[e], xy[e], xl[e], xq[e], n0 + cc) : 0.f;
            }
        } else {
#pragma unroll
            for (int e = 0; e < EPT; ++e) {
                const int idx = e * 256 + t, rr = idx / FK, kk = idx % FK, k = k0 + kk;
                As[kk][rr] = (k < K && m0 + rr < M) ? g_from(xr[e], xy[e], xl[e], xq[e], k) : 0.f;
                Bs[kk][rr] = (k < K && n0 + rr < Nn) ? xa[e] : 0.f;
            }
        }
        if (k0 + FK < K) load_chunk(k0 + FK);
        __syncthreads();
        const int kmax = min(FK, K - k0);   // the chunk's k range (a short last chunk skips its padding)
        if (narrow) {   // at most 16 columns: thread (row nr, column group nc) owns 1 x 4 outputs
#pragma unroll 8
            for (int kk = 0; kk < kmax; ++kk) {
                const float x = As[kk][nr];
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[0][j] = fmaf(x, Bs[kk][nc * 4 + j], acc[0][j]);
            }
        } else {
#pragma unroll 8
            for (int kk = 0; kk < kmax; ++kk) {
                float x[4], w[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) x[i] = As[kk][ty * 4 + i];
#pragma unroll
                for (int j = 0; j < 4; ++j) w[j] = Bs[kk][tx * 4 + j];
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(x[i], w[j], acc[i][j]);
            }
        }
        __syncthreads();
    }
    for (int i = 0; i < (narrow ? 1 : 4); ++i)
        for (int j = 0; j < 4; ++j) {
            const int m = narrow ? m0 + nr : m0 + ty * 4 + i, n = narrow ? n0 + nc * 4 + j : n0 + tx * 4 + j;
            if (m >= M || n >= Nn) continue;
            if (is_dw) {
                float* p = a.dW + (int64_t)m * a.lddw + n;
                *p = a.beta != 0.f ? acc[i][j] + a.beta * *p : acc[i][j];
            } else if (a.dh_bf16) {
                stf<uint16_t>(static_cast<uint16_t*>(a.dH), (int64_t)m * a.lddh + n, acc[i][j]);
            } else {
                stf<float>(static_cast<float*>(a.dH), (int64_t)m * a.lddh + n, acc[i][j]);
            }
        }
    if (blockIdx.x == 0 && a.db != nullptr)
        for (int j = t; j < a.V; j += 256) a.db[j] = nt > 0 ? (1.0f - a.lambda) * a.s[j] + a.lambda * a.q_hat[j] : 0.f;
}

// ---- MFMA bf16 path -----------------------------------------------------------------------------
constexpr int MB = 128;          // output tile (both dims)
constexpr int MK = 64;           // k tile
constexpr int LDK = MK + 8;      // LDS row pitch in bf16 elements (144 bytes)

// Branch-free staging: every 16-byte chunk is loaded unconditionally from a clamped in-range
// address; an out-of-range chunk is zeroed by its lane mask when it is written to LDS (after the
// MFMA phase), so all loads of a tile stay in flight together.
__device__ __forceinline__ uint4 ld16(const uint16_t* p) { return *reinterpret_cast<const uint4*>(p); }

// A tile for dW: A(m, k) = H[k][m], global rows k contiguous in m. Thread t stages k rows
// kq*4..+3 and m columns mq*8..+7 (kq = t / 16, mq = t % 16); transposes with byte permutes.
struct StageHt {
    uint4 r[4];
    uint32_t mk[4];
    __device__ __forceinline__ void load(const uint16_t* H, int64_t ldh, int M, int k0, int kend, int m0) {
        const int t = threadIdx.x, kq = t / 16, mq = t % 16;
        const int m = m0 + mq * 8;
        const bool mok = m < M;
        const int mc = mok ? m : M - 8;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int k = k0 + kq * 4 + q;
            mk[q] = lane_mask(mok && k < kend);
            r[q] = ld16(H + (int64_t)(k < kend ? k : kend - 1) * ldh + mc);
        }
    }
    __device__ __forceinline__ void store(uint16_t (*As)[LDK]) const {
        const int t = threadIdx.x, kq = t / 16, mq = t % 16;
        const uint32_t w0[4] = {r[0].x & mk[0], r[0].y & mk[0], r[0].z & mk[0], r[0].w & mk[0]};
        const uint32_t w1[4] = {r[1].x & mk[1], r[1].y & mk[1], r[1].z & mk[1], r[1].w & mk[1]};
        const uint32_t w2[4] = {r[2].x & mk[2], r[2].y & mk[2], r[2].z & mk[2], r[2].w & mk[2]};
        const uint32_t w3[4] = {r[3].x & mk[3], r[3].y & mk[3], r[3].z & mk[3], r[3].w & mk[3]};
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            // columns m = mq*8 + 2p (low halves) and 2p + 1 (high halves)
            uint2 lo, hi;
            lo.x = __builtin_amdgcn_perm(w1[p], w0[p], 0x05040100u);
            lo.y = __builtin_amdgcn_perm(w3[p], w2[p], 0x05040100u);
            hi.x = __builtin_amdgcn_perm(w1[p], w0[p], 0x07060302u);
            hi.y = __builtin_amdgcn_perm(w3[p], w2[p], 0x07060302u);
            *reinterpret_cast<uint2*>(&As[mq * 8 + 2 * p][kq * 4]) = lo;
            *reinterpret_cast<uint2*>(&As[mq * 8 + 2 * p + 1][kq * 4]) = hi;
        }
    }
};

// B tile for dW: B(k, n) = G(k, n) from R[k][n]; same thread geometry as StageHt, the fold
// G = fma(alpha, R, mask_k * cq_n) in fp32, rounded to bf16 pairs (k, k+1) -- the transpose.
struct StageGt {
    uint4 r[4];
    uint32_t mk[4];
    float vm[4];      // row masks as loaded; rows past kend are dropped by mk at store time
    float zc[4];      // logits input: c of each row and the label's offset in this thread's 8 columns
    int lo[4];
    __device__ __forceinline__ void load(const uint16_t* R, int64_t ldr, int Nn, int k0, int kend, int n0,
                                         const Fold& f) {
        const int t = threadIdx.x, kq = t / 16, mq = t % 16;
        const int n = n0 + mq * 8;
        const bool nok = n < Nn;
        const int nc = nok ? n : Nn - 8;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int k = k0 + kq * 4 + q;
            const int kc = k < kend ? k : kend - 1;
            vm[q] = f.vmask[kc];
            mk[q] = lane_mask(nok && k < kend);
            r[q] = ld16(R + (int64_t)kc * ldr + nc);
            if (f.zc != nullptr) {
                zc[q] = f.zc[kc];
                lo[q] = f.labels[kc] - nc;
            }
        }
    }
    __device__ __forceinline__ void store(uint16_t (*Bs)[LDK], float alpha, const float* cqn, const Fold& f) const {
        const int t = threadIdx.x, kq = t / 16, mq = t % 16;
        uint4 x[4] = {r[0], r[1], r[2], r[3]};
        if (f.zc != nullptr) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const u32x4_t y = z_chunk_to_r(u32x4_t{x[q].x, x[q].y, x[q].z, x[q].w}, zc[q], lo[q], true);
                x[q] = make_uint4(y[0], y[1], y[2], y[3]);
            }
        }
        const uint32_t w[4][4] = {{x[0].x & mk[0], x[0].y & mk[0], x[0].z & mk[0], x[0].w & mk[0]},
                                  {x[1].x & mk[1], x[1].y & mk[1], x[1].z & mk[1], x[1].w & mk[1]},
                                  {x[2].x & mk[2], x[2].y & mk[2], x[2].z & mk[2], x[2].w & mk[2]},
                                  {x[3].x & mk[3], x[3].y & mk[3], x[3].z & mk[3], x[3].w & mk[3]}};
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            float g[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float rv = (c & 1) ? bf16_hi(w[q][c >> 1]) : bf16_lo(w[q][c >> 1]);
                g[q] = fmaf(alpha, rv, vm[q] * cqn[c]);
            }
            uint2 o;
            o.x = pack_bf16x2(g[0], g[1]) & ((mk[0] & 0x0000FFFFu) | (mk[1] & 0xFFFF0000u));
            o.y = pack_bf16x2(g[2], g[3]) & ((mk[2] & 0x0000FFFFu) | (mk[3] & 0xFFFF0000u));
            *reinterpret_cast<uint2*>(&Bs[mq * 8 + c][kq * 4]) = o;
        }
    }
};

// k-contiguous tiles (dH): tile rows are output rows (A) or output columns (B); thread t stages
// rows (e*256 + t) / 8 and k chunk ((e*256 + t) % 8) * 8, e < 4.
template <bool FOLD>
struct StageK {
    uint4 r[4];
    uint32_t mk[4];
    float vm[4];      // FOLD: row masks and the history coefficients of this thread's k chunk, as
    float4 cq[2];     // loaded (consumed at store time, after the MFMA phase)
    float zc[4];      // FOLD with logits input: c of each row and the label's offset in the k chunk
    int lo[4];
    __device__ __forceinline__ void load(const uint16_t* X, int64_t ldx, int rows, int r0, int k0, int kend,
                                         const Fold& f) {
        const int t = threadIdx.x;
        const int k = k0 + (t % 8) * 8;
        const int kc = k < kend ? k : kend - 8;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int c = e * 256 + t, row = r0 + c / 8;
            const int rc = row < rows ? row : rows - 1;
            mk[e] = lane_mask(row < rows && k < kend);
            r[e] = ld16(X + (int64_t)rc * ldx + kc);
            if (FOLD) vm[e] = f.vmask[rc];
            if (FOLD && f.zc != nullptr) {
                zc[e] = f.zc[rc];
                lo[e] = f.labels[rc] - kc;
            }
        }
        if (FOLD) {
            cq[0] = *reinterpret_cast<const float4*>(f.cq + kc);
            cq[1] = *reinterpret_cast<const float4*>(f.cq + kc + 4);
        }
    }
    __device__ __forceinline__ void store(uint16_t (*S)[LDK], float alpha, const Fold& f) const {
        const int t = threadIdx.x;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int c = e * 256 + t, lr = c / 8, lk = (c % 8) * 8;
            uint4 o = r[e];
            if (FOLD && f.zc != nullptr) {
                const u32x4_t x = z_chunk_to_r(u32x4_t{o.x, o.y, o.z, o.w}, zc[e], lo[e], true);
                o = make_uint4(x[0], x[1], x[2], x[3]);
            }
            if (FOLD) {
                const float q8[8] = {cq[0].x, cq[0].y, cq[0].z, cq[0].w, cq[1].x, cq[1].y, cq[1].z, cq[1].w};
                const uint32_t w[4] = {o.x, o.y, o.z, o.w};
                uint32_t g[4];
#pragma unroll
                for (int p = 0; p < 4; ++p)
                    g[p] = pack_bf16x2(fmaf(alpha, bf16_lo(w[p]), vm[e] * q8[2 * p]),
                                       fmaf(alpha, bf16_hi(w[p]), vm[e] * q8[2 * p + 1]));
                o = make_uint4(g[0], g[1], g[2], g[3]);
            }
            *reinterpret_cast<uint4*>(&S[lr][lk]) = and_mask(o, mk[e]);
        }
    }
};

__device__ __forceinline__ void mfma_tile(const uint16_t (*As)[LDK], const uint16_t (*Bs)[LDK], f32x16_t (&acc)[2][2]) {
    const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
    const int wm = w / 2, wn = w % 2;
    const int lr = lane % 32, lk = (lane / 32) * 8;
#pragma unroll
    for (int kk = 0; kk < MK; kk += 16) {
        bf16x8_t a[2], b[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) a[i] = *reinterpret_cast<const bf16x8_t*>(&As[wm * 64 + i * 32 + lr][kk + lk]);
#pragma unroll
        for (int j = 0; j < 2; ++j) b[j] = *reinterpret_cast<const bf16x8_t*>(&Bs[wn * 64 + j * 32 + lr][kk + lk]);
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
}

// Accumulator element r of lane l in block (i, j) sits at tile row wm*64 + i*32 + (r/4)*8 + (l/32)*4 + r%4
// and tile column wn*64 + j*32 + l%32.
template <typename F>
__device__ __forceinline__ void for_each_acc(const f32x16_t (&acc)[2][2], F&& fn) {
    const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
    const int wm = w / 2, wn = w % 2;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                fn(wm * 64 + i * 32 + (r / 4) * 8 + (lane / 32) * 4 + (r % 4), wn * 64 + j * 32 + lane % 32, acc[i][j][r]);
}

// k tiles a 128-tile workgroup loads at once when its k range is short (the latency-bound regime
// of small products): one round trip to memory, then the tiles go through LDS one after another.
constexpr int kPre = 4;

// Shared k loop of the 128-tile kernels. LA / LB load operand tiles into staging registers,
// SA / SB write them to an LDS buffer.
template <typename StA, typename StB, typename LA, typename LB, typename SA, typename SB>
__device__ __forceinline__ void k_loop128(int kb, int ke, uint16_t (*As)[MB][LDK], uint16_t (*Bs)[MB][LDK],
                                          f32x16_t (&acc)[2][2], LA&& load_a, LB&& load_b, SA&& store_a,
                                          SB&& store_b) {
    const int nk = (ke - kb + MK - 1) / MK;
    if (nk <= kPre) {
        StA sa[kPre];
        StB sb[kPre];
#pragma unroll
        for (int q = 0; q < kPre; ++q) {   // tiles past ke load clamped rows and stage zeros
            load_a(sa[q], kb + q * MK);
            load_b(sb[q], kb + q * MK);
        }
#pragma unroll
        for (int q = 0; q < kPre; ++q) {
            if (q < nk) {   // uniform
                store_a(sa[q], As[q & 1]);
                store_b(sb[q], Bs[q & 1]);
                __syncthreads();   // also: every wave is done with the buffer's previous tile
                mfma_tile(As[q & 1], Bs[q & 1], acc);
            }
        }
        return;
    }
    StA sa;
    StB sb;
    load_a(sa, kb);
    load_b(sb, kb);
    store_a(sa, As[0]);
    store_b(sb, Bs[0]);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        const bool more = kt + 1 < nk;
        if (more) {
            load_a(sa, kb + (kt + 1) * MK);
            load_b(sb, kb + (kt + 1) * MK);
        }
        mfma_tile(As[buf], Bs[buf], acc);
        if (more) {
            store_a(sa, As[buf ^ 1]);
            store_b(sb, Bs[buf ^ 1]);
        }
        __syncthreads();
    }
}

// dW[m][n] = sum_k H[k][m] G[k][n]: M = d, Nn = V, K = N rows.
__global__ __launch_bounds__(256) void mfma_dW_kernel(const uint16_t* __restrict__ H, int64_t ldh,
                                                      const uint16_t* __restrict__ R, int64_t ldr, int M, int Nn, int K,
                                                      int kps, Fold f, float* __restrict__ out, int64_t ldo, float beta,
                                                      float* __restrict__ part) {
    __shared__ __attribute__((aligned(16))) uint16_t As[2][MB][LDK];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[2][MB][LDK];
    const int m0 = blockIdx.y * MB, n0 = blockIdx.x * MB;
    const int kb = blockIdx.z * kps, ke = min(K, kb + kps);
    const float alpha = f.scal[0];
    float cqn[8];
    {
        const int n = n0 + (threadIdx.x % 16) * 8;
#pragma unroll
        for (int c = 0; c < 8; ++c) cqn[c] = (n + c < Nn) ? f.cq[n + c] : 0.f;
    }
    f32x16_t acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    k_loop128<StageHt, StageGt>(
        kb, ke, As, Bs, acc, [&](StageHt& st, int k0) { st.load(H, ldh, M, k0, ke, m0); },
        [&](StageGt& st, int k0) { st.load(R, ldr, Nn, k0, ke, n0, f); },
        [&](const StageHt& st, uint16_t (*S)[LDK]) { st.store(S); },
        [&](const StageGt& st, uint16_t (*S)[LDK]) { st.store(S, alpha, cqn, f); });
    if (part == nullptr) {
        for_each_acc(acc, [&](int r, int c, float v) {
            const int m = m0 + r, n = n0 + c;
            if (m < M && n < Nn) {
                float* p = out + (int64_t)m * ldo + n;
                *p = beta != 0.f ? v + beta * *p : v;
            }
        });
    } else {
        float* pz = part + (int64_t)blockIdx.z * M * Nn;
        for_each_acc(acc, [&](int r, int c, float v) {
            const int m = m0 + r, n = n0 + c;
            if (m < M && n < Nn) pz[(int64_t)m * Nn + n] = v;
        });
    }
}

// dH[i][n] = sum_j G[i][j] W[n][j]: M = N rows, Nn = d, K = V.
template <typename TO>
__global__ __launch_bounds__(256) void mfma_dH_kernel(const uint16_t* __restrict__ R, int64_t ldr,
                                                      const uint16_t* __restrict__ W, int64_t ldw, int M, int Nn, int K,
                                                      int kps, Fold f, TO* __restrict__ out, int64_t ldo,
                                                      float* __restrict__ part) {
    __shared__ __attribute__((aligned(16))) uint16_t As[2][MB][LDK];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[2][MB][LDK];
    const int m0 = blockIdx.y * MB, n0 = blockIdx.x * MB;
    const int kb = blockIdx.z * kps, ke = min(K, kb + kps);
    const float alpha = f.scal[0];
    f32x16_t acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    k_loop128<StageK<true>, StageK<false>>(
        kb, ke, As, Bs, acc, [&](StageK<true>& st, int k0) { st.load(R, ldr, M, m0, k0, ke, f); },
        [&](StageK<false>& st, int k0) { st.load(W, ldw, Nn, n0, k0, ke, f); },
        [&](const StageK<true>& st, uint16_t (*S)[LDK]) { st.store(S, alpha, f); },
        [&](const StageK<false>& st, uint16_t (*S)[LDK]) { st.store(S, alpha, f); });
    if (part == nullptr) {
        for_each_acc(acc, [&](int r, int c, float v) {
            const int m = m0 + r, n = n0 + c;
            if (m < M && n < Nn) stf<TO>(out, (int64_t)m * ldo + n, v);
        });
    } else {
        float* pz = part + (int64_t)blockIdx.z * M * Nn;
        for_each_acc(acc, [&](int r, int c, float v) {
            const int m = m0 + r, n = n0 + c;
            if (m < M && n < Nn) pz[(int64_t)m * Nn + n] = v;
        });
    }
}

// ---- MFMA bf16, 256 x 256 tiles: shared helpers ---------------------------------------------------
// LDS rows of 64 bf16 (128 B, no padding): the 16-byte chunk c of row r lives at chunk
// c ^ ((r ^ (r >> 3)) & 7), free of bank conflicts on gfx950 for 16-byte fragment reads and for the
// 1 KB-per-wave staging writes.
__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row ^ (row >> 3)) & 7); }

template <typename F>
__device__ __forceinline__ void for_each_acc256(const f32x16_t (&acc)[4][4], F&& fn) {
    const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
    const int wm = w / 2, wn = w % 2;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                fn(wm * 128 + i * 32 + (r / 4) * 8 + (lane / 32) * 4 + (r % 4), wn * 128 + j * 32 + lane % 32,
                   acc[i][j][r]);
}

// Workgroup -> tile map: tiles along the short dimension ("inner", reused operand) that share a
// long-dimension tile run on one XCD together (workgroups are dealt to the 8 XCDs round-robin).
__device__ __forceinline__ bool tile_of(int inner_count, int outer_count, bool inner_is_m, int* tm, int* tn) {
    const int id = blockIdx.x;
    const int xcd = id % 8, rest = id / 8;
    const int inner = rest % inner_count, og = rest / inner_count;
    const int outer = og * 8 + xcd;
    if (outer >= outer_count) return false;
    *tm = inner_is_m ? inner : outer;
    *tn = inner_is_m ? outer : inner;
    return true;
}

// A launch over the outer tiles [outer_begin, outer_end), each split into `splits` k ranges (whole
// rounds of the chip run with the full k range; the leftover tiles split k so that they fill the chip
// too). Split partials go to a rectangle of fp32 sums with origin (pm0, pn0), leading dimension ldp and
// split stride pstride.
struct TileRange {
    int inner_count, outer_begin, outer_end, splits;
    int pm0, pn0;
    int64_t ldp, pstride;
    int blocked;   // 1: an XCD's 32 concurrent tiles are 4 outer x 8 inner (needs splits = 1, inner_count % 8 = 0)
};

// Work unit of this workgroup. The pairs (outer tile, k split) are dealt to the 8 XCDs round-robin
// (workgroups are dealt to the XCDs round-robin by id), and all inner tiles of a pair run on the same
// XCD, so the tiles that share an outer operand panel share that XCD's L2. With one split this is the
// plain outer-tile order: XCD x runs outer tiles x, x + 8, x + 16, ...
// Blocked order (r.blocked): with more than 8 inner tiles, the 32 tiles an XCD runs at once are 4 of its
// outer tiles x 8 inner tiles instead of 2 outer tiles x all inner tiles; the XCD's L2 then misses on 12
// operand panels per round instead of 2 + inner_count (18 at 16 inner tiles). XCD x still owns the outer
// tiles x, x + 8, ...; it takes them 4 at a time (the last group may be shorter) and runs each group's
// inner tiles 8 at a time.
__device__ __forceinline__ bool unit_of(const TileRange& r, bool inner_is_m, int id, int* tm, int* tn, int* z) {
    const int xcd = id % 8, rest = id / 8;
    if (r.blocked) {
        constexpr int GO = 4, GI = 8;
        const int I = r.inner_count;
        const int lx = (r.outer_end - r.outer_begin - xcd + 7) / 8;   // outer tiles owned by this XCD
        if (rest >= lx * I) return false;
        const int g0 = rest / (GO * I) * GO;                          // first owned outer tile of the group
        const int gsz = min(GO, lx - g0);
        const int within = rest - g0 * I;                             // < gsz * I
        const int ig = within / (gsz * GI), w2 = within % (gsz * GI);
        const int outer = r.outer_begin + xcd + 8 * (g0 + w2 / GI);
        const int inner = ig * GI + w2 % GI;
        *z = 0;
        *tm = inner_is_m ? inner : outer;
        *tn = inner_is_m ? outer : inner;
        return true;
    }
    const int inner = rest % r.inner_count, pg = rest / r.inner_count;
    const int pair = pg * 8 + xcd;
    if (pair >= (r.outer_end - r.outer_begin) * r.splits) return false;
    const int outer = r.outer_begin + pair / r.splits;
    *z = pair % r.splits;
    *tm = inner_is_m ? inner : outer;
    *tn = inner_is_m ? outer : inner;
    return true;
}

// C[m][n] = sum_k A(m, k) B(k, n) for dW (A = H^T k-contiguous, B = G from R) or dH (A = G from R,
// B = W). Output fp32 (with beta) or TO, or fp32 split-K partials.
// ---- MFMA bf16, rank-1 form -----------------------------------------------------------------------
// Rank-1 form of the fold: with alpha = (1 - lambda) / N_t and rows of R outside I equal to zero,
//   dW = alpha H^T R + hsum cq^T,   hsum_m = sum_{i in I} H_im,  cq_n = lambda q_hat_n / N_t,
//   dH = alpha R W^T + mask u^T,    u_n = (lambda / N_t) sum_j W_nj q_hat_j,
// so both GEMMs take R as it is stored (bf16, no rounding of G) and the history enters through
// the fp32 epilogue. 256 x 256 output tile per workgroup, on v_mfma_f32_32x32x16_bf16: eight waves of
// 128 x 64 (or four of 128 x 128). Memory reads are buffer loads: a chunk outside the matrix
// reads as zero through the descriptor's range check or an out-of-range offset, so loads need no
// branches and never touch memory past the operand.
constexpr int LB = 256;                 // output tile


typedef short v4s_t __attribute__((ext_vector_type(4)));
typedef short v8s_t __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) v4s_t lds_v4s_t;

__device__ __forceinline__ bf16x8_t ld_frag_b128(const char* p) { return *reinterpret_cast<const bf16x8_t*>(p); }

__device__ __forceinline__ bf16x8_t ld_frag_tr(const char* p) {
    const v4s_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t*)(p));
    const v4s_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t*)(p + 4 * 512));
    const v8s_t both = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8_t, both);
}

// C = A B for one 256 x 256 output tile over k in [kb, ke), k tiles of 64 in two LDS stages (one barrier
// per 64 k): the workgroup copies 32 kilobytes per operand per tile, 1 KB per wave and copy step, with
// buffer loads into registers and ds_write_b128 (copies straight from memory into LDS with buffer_load
// ... lds share the same ~64 B/clk LDS fill bandwidth and measured slower). A k-contiguous operand (dH's
// two) has LDS rows of 64 k (128 B) with chunk c of row r at swz(r, c) and 16-byte fragment reads; a
// k-outer operand (dW's two) has LDS rows of 256 values per k (512 B), chunk c of row k at
// c ^ ((k & 3) << 2), and fragments read with the transposing ds_read_b64_tr_b16 (a 16-lane group reads a
// 4 x 16 block and each lane receives 4 consecutive k of one column); every 16-lane read phase touches
// 16 distinct 16-byte bank groups, so there are no bank conflicts. (dW with A given as H^T, k-contiguous, from a transpose of H measured no
// faster: the transposing reads of one operand are not what bounds it.) Tile kt+1 is written from registers at the start of
// iteration kt and tile kt+2 loaded behind it; the barrier sits before the last MFMA step of the tile.
// Measured on the three language-model shapes, eight waves (two per SIMD) beat four by 5-9 % on every
// product: with one wave per SIMD the copies, LDS writes and fragment reads add to the MFMA time almost
// in full (removing each of them from a four-wave copy of the kernel saved 14 %, 10 % and 12 % at the
// 1B shape), while a second wave issues its MFMAs meanwhile, at the price of 1.5 x the fragment reads.
constexpr int WKT = 64;             // k tile of the 64-deep kernels
constexpr int WSE = LB * WKT;        // bf16 elements per operand per stage (32 KB)

// Arguments of one 64-deep 256-tile product (one launch part).
struct WideArgs {
    const uint16_t* Xa;
    int64_t lda;
    const uint16_t* Xb;
    int64_t ldb;
    int M, Nn, K, kps;
    TileRange tr;
    const float* alpha_p;
    const float* rv;
    const float* cv;
    void* out;
    int64_t ldo;
    float beta;
    float* part;
    const uint16_t* bias;   // forward: bf16 bias [Nn] or null
    const float* zc;        // logits input (ZR): c_i per row of R, and the labels
    const int32_t* labels;
    // forward with row statistics: per (row, 256-column tile) records (max, sum of exp(z - max), first
    // argmax) of the rounded logits at stats + (row * stats_ld + tile) * 3, and the target logit of each
    // row whose label is valid (written by the tile that holds the label)
    float* stats;
    int64_t stats_ld;
    int32_t ignore_index;
    float* row_target;
};

// Products of the 64-deep kernel: C = A B with
//   kWideDH:  dH = alpha R W^T + rv cv^T     A(m, k) = R[m][k], B(k, n) = W[n][k] (both k-contiguous)
//   kWideDW:  dW = alpha H^T R + rv cv^T (+ beta dW)   A(m, k) = H[k][m], B(k, n) = R[k][n] (both k-outer)
//   kWideFWD: Z = H W (+ b)                  A(m, k) = H[m][k] (k-contiguous), B(k, n) = W[k][n] (k-outer)
constexpr int kWideDH = 0, kWideDW = 1, kWideFWD = 2;

// One work unit (tile and k range) of the product, for block id `id` of its launch part; lds and rv_s
// are the workgroup's LDS (two stages of both operands, and the rank-1 row vector of the tile).
// NW waves share the 256 x 256 tile: four (one per SIMD) each own 128 x 128, or eight (two per SIMD,
// so that one wave's copies and LDS reads overlap the other's MFMAs) each own 128 x 64.
// ZR: the operand that is R (dH's A, dW's B) holds the logits Z, and each copy is turned into R in
// registers before its LDS write (z_chunk_to_r).
template <int MODE, typename TO, int NW, bool ZR = false, bool FS = false>
__device__ __forceinline__ void wide_tile(const WideArgs& args, int id, uint16_t (&lds)[2][2][WSE], float (&rv_s)[LB],
                                          float2* zs = nullptr) {
    static_assert(NW == 4 || NW == 8, "four or eight waves");
    constexpr int KT = WKT;
    constexpr int WCOLS = NW == 4 ? 128 : 64;   // columns of a wave's part of the tile
    constexpr int NJ = WCOLS / 32;              // 32-column MFMA blocks per wave
    constexpr int CPO = 32 / NW;                // 1 KB copy steps per operand per k tile, per wave
    constexpr int CPS = 2 * CPO < 8 ? 2 * CPO : 8;   // copy steps placed in each of the first MFMA steps
    constexpr bool IS_DW = MODE == kWideDW;
    constexpr bool RANK1 = MODE != kWideFWD;   // rank-1 epilogue (the head VJP products)
    constexpr bool KA = MODE != kWideDW;       // operand A k-contiguous
    constexpr bool KB = MODE == kWideDH;       // operand B k-contiguous
    const uint16_t* __restrict__ Xa = args.Xa;
    const int64_t lda = args.lda;
    const uint16_t* __restrict__ Xb = args.Xb;
    const int64_t ldb = args.ldb;
    const int M = args.M, Nn = args.Nn, K = args.K, kps = args.kps;
    const TileRange& tr = args.tr;
    const float* alpha_p = args.alpha_p;
    const float* __restrict__ rv = args.rv;
    const float* __restrict__ cv = args.cv;
    TO* __restrict__ out = static_cast<TO*>(args.out);
    const int64_t ldo = args.ldo;
    const float beta = args.beta;
    float* __restrict__ part = args.part;
    int tm, tn, kz;
    if (!unit_of(tr, MODE != kWideDH, id, &tm, &tn, &kz)) return;
    // uniform per workgroup: keep them scalar so that the buffer descriptors stay in SGPRs
    tm = __builtin_amdgcn_readfirstlane(tm);
    tn = __builtin_amdgcn_readfirstlane(tn);
    kz = __builtin_amdgcn_readfirstlane(kz);
    const int m0 = tm * LB, n0 = tn * LB;
    const int kb = kz * kps, ke = min(K, kb + kps);
    const int nk = (ke - kb + KT - 1) / KT;
    const int l = threadIdx.x % kWave;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int wm = wave / (NW / 2), wn = wave % (NW / 2);

    // rank-1 term of the epilogue (none when rv is null: lambda = 0 has no history term)
    const bool r1 = RANK1 && part == nullptr && rv != nullptr;
    const float rv_reg = (r1 && (int)threadIdx.x < LB && m0 + (int)threadIdx.x < M) ? rv[m0 + threadIdx.x] : 0.f;
    float cvv[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int n = n0 + wn * WCOLS + j * 32 + l % 32;
        cvv[j] = (r1 && n < Nn) ? cv[n] : 0.f;
    }

    // copy step q (< CPO) of this wave fills kilobyte wave*CPO + q of an operand's stage
    int voff_a[CPO], voff_b[CPO], kc_a[CPO], kc_b[CPO];
    bool ok_a[CPO], ok_b[CPO];
    auto geo = [&](bool kcontig, int64_t ld, int rows_valid, int q, int* voff, int* kc, bool* ok) {
        const int chunk = (wave * CPO + q) * 64 + l;
        if (kcontig) {
            const int row = chunk / 8, c = swz(row, chunk % 8);
            *voff = (int)((int64_t)row * ld * 2) + c * 16;
            *kc = c * 8;
            *ok = row < rows_valid;
        } else {
            const int krow = chunk / 32, c = (chunk % 32) ^ ((krow & 3) << 2);
            *voff = (int)((int64_t)krow * ld * 2) + c * 16;
            *kc = krow;
            *ok = true;
        }
    };
#pragma unroll
    for (int q = 0; q < CPO; ++q) {
        geo(KA, lda, M - m0, q, &voff_a[q], &kc_a[q], &ok_a[q]);
        geo(KB, ldb, Nn - n0, q, &voff_b[q], &kc_b[q], &ok_b[q]);
    }
    // logits input: c of each row of the R operand and its label. dH: the tile's 256 rows are fixed, so
    // (c, label) sit in LDS (zs) and each copy looks its row up at write time, the label as an offset
    // from the chunk's k; dW: rows change with the k tile, so both are loaded into registers with each
    // copy, the label as an offset from the chunk's first column
    constexpr bool ZA = ZR && MODE == kWideDH, ZB = ZR && MODE == kWideDW;
    float zrc[CPO];
    int zry[CPO], zcol[CPO];
#pragma unroll
    for (int q = 0; q < CPO; ++q) {
        zrc[q] = INFINITY;
        zry[q] = -1;
        zcol[q] = 0;
        const int chunk = (wave * CPO + q) * 64 + l;
        if constexpr (ZB) zcol[q] = n0 + (((chunk % 32) ^ (((chunk / 32) & 3) << 2)) << 3);
    }
    // k-contiguous operands: one descriptor per workgroup over the tile's rows (exact extent)
    const int bytes_ta = KA ? (int)(((int64_t)(min(LB, M - m0) - 1) * lda + K) * 2) : 0;
    const int bytes_tb = KB ? (int)(((int64_t)(min(LB, Nn - n0) - 1) * ldb + K) * 2) : 0;
    struct TileLoad {
        const uint16_t* ba;
        const uint16_t* bb;
        int bytes_a, bytes_b, k0;
    };
    // k-outer operands: descriptors rebased on (k0, first column) per k tile, rows at or past ke read zeros
    auto tile_load = [&](int kt) {
        TileLoad tl;
        tl.k0 = kb + kt * KT;
        const int nv = min(KT, ke - tl.k0);
        const int nv1 = max(nv, 1);
        const int kr = min(tl.k0, K - 1);
        if constexpr (KA) {
            tl.ba = Xa + (int64_t)m0 * lda;
            tl.bytes_a = bytes_ta;
        } else {
            tl.ba = Xa + (int64_t)kr * lda + m0;
            tl.bytes_a = nv > 0 ? (int)(((int64_t)(nv1 - 1) * lda + (M - m0)) * 2) : 0;
        }
        if constexpr (KB) {
            tl.bb = Xb + (int64_t)n0 * ldb;
            tl.bytes_b = bytes_tb;
        } else {
            tl.bb = Xb + (int64_t)kr * ldb + n0;
            tl.bytes_b = nv > 0 ? (int)(((int64_t)(nv1 - 1) * ldb + (Nn - n0)) * 2) : 0;
        }
        return tl;
    };
    // copy op q < 2 CPO: q < CPO operand A, else operand B
    auto load_one = [&](const TileLoad& tl, int q) {
        if (q < CPO) {
            const int vo = !KA ? voff_a[q] : ((ok_a[q] && tl.k0 + kc_a[q] < ke) ? voff_a[q] + tl.k0 * 2 : kOob);
            return __builtin_amdgcn_raw_buffer_load_b128(make_desc(tl.ba, tl.bytes_a), vo, 0, 0);
        }
        const int r = q - CPO;
        if constexpr (ZB) {   // the row of this copy: its c and its label's offset from the chunk's columns
            const int k = tl.k0 + kc_b[r];
            const bool kin = k < ke;
            const int kcl = kin ? k : K - 1;
            zrc[r] = kin ? args.zc[kcl] : INFINITY;
            zry[r] = kin ? args.labels[kcl] - zcol[r] : -1;
        }
        const int vo = !KB ? voff_b[r] : ((ok_b[r] && tl.k0 + kc_b[r] < ke) ? voff_b[r] + tl.k0 * 2 : kOob);
        return __builtin_amdgcn_raw_buffer_load_b128(make_desc(tl.bb, tl.bytes_b), vo, 0, 0);
    };
    // k0w: the first k of the tile whose copy v holds
    auto write_one = [&](int stage, int q, const u32x4_t& v, int k0w) {
        char* base = reinterpret_cast<char*>(&lds[stage][q / CPO][0]);
        u32x4_t x = v;
        if constexpr (ZA) {
            if (q < CPO) {
                const int j0 = k0w + kc_a[q];
                const float2 zz = zs[((wave * CPO + q) * 64 + l) / 8];   // the copy's row: c and label
                x = z_chunk_to_r(v, zz.x, __float_as_int(zz.y) - j0, ok_a[q] && j0 < ke);
            }
        }
        if constexpr (ZB) {
            if (q >= CPO) x = z_chunk_to_r(v, zrc[q - CPO], zry[q - CPO], true);
        }
        *reinterpret_cast<u32x4_t*>(base + (wave * CPO + q % CPO) * 1024 + l * 16) = x;
    };

    // fragments for MFMA step s (k = 16 s .. +15) of `cnt` 32-wide blocks from tile row/column `base`:
    // k-outer offsets (transposing reads; the 16-byte chunk of a k row is swizzled by (k & 3) << 2) or
    // LDS rows (16-byte reads; the chunk depends on the step)
    int fa[4], fb[NJ];
    auto frag_geo = [&](bool kcontig, int base, int cnt, int* f) {
        if (kcontig) {
#pragma unroll
            for (int i = 0; i < cnt; ++i) f[i] = base + i * 32 + l % 32;
        } else {
            const int s = l % 16, g = l / 16;
            const int krow = (g >> 1) * 8 + (s >> 2);
#pragma unroll
            for (int i = 0; i < cnt; ++i) {
                const int chunk = ((base / 8 + i * 4) ^ ((krow & 3) << 2)) + (g & 1) * 2 + ((s >> 1) & 1);
                f[i] = krow * 512 + (chunk << 4) + (s & 1) * 8;
            }
        }
    };
    frag_geo(KA, wm * 128, 4, fa);
    frag_geo(KB, wn * WCOLS, NJ, fb);
    auto read_frags = [&](int stage, int s, bf16x8_t (&a)[4], bf16x8_t (&b)[NJ]) {
        const char* As = reinterpret_cast<const char*>(&lds[stage][0][0]);
        const char* Bs = reinterpret_cast<const char*>(&lds[stage][1][0]);
        const int c = 2 * s + l / 32;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if constexpr (KA) a[i] = ld_frag_b128(As + fa[i] * 128 + swz(fa[i], c) * 16);
            else a[i] = ld_frag_tr(As + fa[i] + s * 16 * 512);
        }
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            if constexpr (KB) b[j] = ld_frag_b128(Bs + fb[j] * 128 + swz(fb[j], c) * 16);
            else b[j] = ld_frag_tr(Bs + fb[j] + s * 16 * 512);
        }
    };

    f32x16_t acc[4][NJ];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    // one MFMA step; copy ops q0 .. q0+CPS-1 placed after its first MFMAs (if q0 >= 0)
    auto step = [&](const bf16x8_t (&a)[4], const bf16x8_t (&b)[NJ], int q0, int ws, const TileLoad& tl,
                    u32x4_t (&rg)[2 * CPO]) {
#pragma unroll
        for (int m = 0; m < 4 * NJ; ++m) {
            acc[m / NJ][m % NJ] =
                __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[m / NJ], b[m % NJ], acc[m / NJ][m % NJ], 0, 0, 0);
            if (q0 >= 0 && m < CPS) {
                __builtin_amdgcn_sched_barrier(0);
                write_one(ws, q0 + m, rg[q0 + m], tl.k0 - KT);
                rg[q0 + m] = load_one(tl, q0 + m);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    };
    // scheduling of a step without copies: the next step's fragment reads (issued before the step)
    // spread one group after each MFMA instead of ahead of them all
    constexpr int kReads = (KA ? 4 : 8) + (KB ? NJ : 2 * NJ);   // LDS read instructions per step
    constexpr int kRpm = (kReads + 7) / 8;
    auto spread_reads = [&]() {
#pragma unroll
        for (int q = 0; q < kReads / kRpm; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);      // MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, kRpm, 0);   // LDS read
        }
        __builtin_amdgcn_sched_group_barrier(0x008, 4 * NJ - kReads / kRpm, 0);
    };
    u32x4_t rg[2 * CPO];
    bf16x8_t a0[4], b0[NJ], a1[4], b1[NJ];
    if constexpr (ZA) {   // logits rows of the tile: c and label, held in LDS (registers are taken in full)
        for (int t = threadIdx.x; t < LB; t += NW * kWave) {
            const int i = m0 + t;
            zs[t] = i < M ? make_float2(args.zc[i], __int_as_float(args.labels[i])) : make_float2(INFINITY, __int_as_float(-1));
        }
        __syncthreads();
    }
    {
        const TileLoad t0 = tile_load(0), t1 = tile_load(1);
#pragma unroll
        for (int q = 0; q < 2 * CPO; ++q) rg[q] = load_one(t0, q);
#pragma unroll
        for (int q = 0; q < 2 * CPO; ++q) write_one(0, q, rg[q], t0.k0);
#pragma unroll
        for (int q = 0; q < 2 * CPO; ++q) rg[q] = load_one(t1, q);
    }
    __syncthreads();
    read_frags(0, 0, a0, b0);
    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1, nxt = cur ^ 1;
        const TileLoad tl = tile_load(kt + 2);
        read_frags(cur, 1, a1, b1);
        step(a0, b0, 0, nxt, tl, rg);
        __builtin_amdgcn_sched_barrier(0);
        read_frags(cur, 2, a0, b0);
        step(a1, b1, 2 * CPO > CPS ? CPS : -1, nxt, tl, rg);
        if constexpr (2 * CPO <= CPS) spread_reads();
        __builtin_amdgcn_sched_barrier(0);
        read_frags(cur, 3, a1, b1);
        step(a0, b0, -1, nxt, tl, rg);
        spread_reads();
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        __builtin_amdgcn_sched_barrier(0);
        read_frags(nxt, 0, a0, b0);
        step(a1, b1, -1, nxt, tl, rg);
        spread_reads();
        __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
    // accumulator element (i, j, r) of this lane: tile row and column, and the 32-column block j
    auto for_each_acc = [&](auto&& fn) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < NJ; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    fn(wm * 128 + i * 32 + (r / 4) * 8 + (l / 32) * 4 + (r % 4), wn * WCOLS + j * 32 + l % 32, j,
                       acc[i][j][r]);
    };
    if constexpr (MODE == kWideFWD) {
        const uint16_t* __restrict__ bias = args.bias;
        if constexpr (!FS) {
            for_each_acc([&](int r, int c, int, float v) {
                const int m = m0 + r, n = n0 + c;
                if (m < M && n < Nn) stf<TO>(out, (int64_t)m * ldo + n, bias ? v + bf16_to_f32(bias[n]) : v);
            });
            return;
        } else if constexpr (std::is_same<TO, uint16_t>::value) {
            // row statistics: the rounded tile goes to LDS (the operand stages are free after the k loop:
            // 256 rows of 512 bytes), then two threads per row store it with 16-byte writes and reduce
            // their 128 columns (maximum, first column reaching it, sum of exp(z - max)); the pair's
            // records are merged and the row's record for this tile is written
            // 16-byte chunk c8 of row r sits at chunk c8 ^ (r % 32): the two threads of each row read
            // 32 different chunk positions across a wave, so the reads are free of bank conflicts
            uint16_t* zt = &lds[0][0][0];
            auto zpos = [](int r, int c) { return r * LB + ((((c >> 3) ^ (r & 31))) << 3) + (c & 7); };
            for_each_acc([&](int r, int c, int, float v) {
                const float x = bias && n0 + c < Nn ? v + bf16_to_f32(bias[n0 + c]) : v;
                zt[zpos(r, c)] = f32_to_bf16(x);
            });
            __syncthreads();
            const int t = threadIdx.x;
            for (int rr = t / 2; rr < LB; rr += NW * 32) {
                const int h = t % 2;
                const int m = m0 + rr;
                const int ncol = min(128, Nn - n0 - h * 128);   // columns of this half inside the matrix
                // pass 1: store the chunks, maximum and its first column (columns past the matrix: -inf)
                float mx = -INFINITY;
                int am = 0;
                uint4 wk[16];
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    const int c = h * 128 + q * 8;
                    wk[q] = *reinterpret_cast<const uint4*>(zt + zpos(rr, c));
                    if (m < M && q * 8 < ncol)
                        *reinterpret_cast<uint4*>(static_cast<uint16_t*>(args.out) + (int64_t)m * ldo + n0 + c) = wk[q];
                    const uint32_t ww[4] = {wk[q].x, wk[q].y, wk[q].z, wk[q].w};
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        const float x = q * 8 + k < ncol ? ((k & 1) ? bf16_hi(ww[k / 2]) : bf16_lo(ww[k / 2])) : -INFINITY;
                        am = x > mx ? c + k : am;
                        mx = fmaxf(mx, x);
                    }
                }
                am += n0;
                // pass 2: sum of exp(z - max) (padding contributes 0)
                const float mx2 = mx * kLog2e;
                float sum = 0.f;
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    const uint32_t ww[4] = {wk[q].x, wk[q].y, wk[q].z, wk[q].w};
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        const float x = q * 8 + k < ncol ? ((k & 1) ? bf16_hi(ww[k / 2]) : bf16_lo(ww[k / 2])) : -INFINITY;
                        sum += exp2_fast(fmaf(x, kLog2e, -mx2));
                    }
                }
                // merge with the other half of the row (lane t ^ 1); the lower columns win ties
                const float mo = __shfl_xor(mx, 1, kWave), so = __shfl_xor(sum, 1, kWave);
                const int ao = __shfl_xor(am, 1, kWave);
                if (h == 0 && m < M) {
                    float M2 = mx, S2 = sum;
                    int A2 = am;
                    if (mo > mx) {
                        S2 = (mx == -INFINITY ? 0.f : sum * exp2_fast((mx - mo) * kLog2e)) + so;
                        M2 = mo;
                        A2 = ao;
                    } else if (mo != -INFINITY) {
                        S2 = sum + so * exp2_fast((mo - mx) * kLog2e);
                    }
                    float* rec = args.stats + ((int64_t)m * args.stats_ld + tn) * 3;
                    rec[0] = M2;
                    rec[1] = S2;
                    rec[2] = __int_as_float(A2);
                    const int y = args.labels[m];
                    if (y != args.ignore_index && y >= n0 && y < n0 + LB && y < Nn)
                        args.row_target[m] = bf16_to_f32(zt[zpos(rr, y - n0)]);
                }
            }
        }
        return;
    }
    const float alpha = *alpha_p;
    if (part == nullptr) {
        if ((int)threadIdx.x < LB) rv_s[threadIdx.x] = rv_reg;
        __syncthreads();
        for_each_acc([&](int r, int c, int j, float v) {
            const int m = m0 + r, n = n0 + c;
            if (m < M && n < Nn) {
                const float x = fmaf(alpha, v, rv_s[r] * cvv[j]);
                if constexpr (IS_DW) {
                    float* p = reinterpret_cast<float*>(out) + (int64_t)m * ldo + n;
                    *p = beta != 0.f ? x + beta * *p : x;
                } else {
                    stf<TO>(out, (int64_t)m * ldo + n, x);
                }
            }
        });
    } else {
        float* pz = part + (int64_t)kz * tr.pstride;
        for_each_acc([&](int r, int c, int, float v) {
            const int m = m0 + r, n = n0 + c;
            if (m < M && n < Nn) pz[(int64_t)(m - tr.pm0) * tr.ldp + (n - tr.pn0)] = alpha * v;
        });
    }
}

template <bool IS_DW, typename TO, int NW, bool ZR = false>
__global__ __launch_bounds__(NW * 64, 1) void lds256w_kernel(WideArgs a) {
    __shared__ __attribute__((aligned(1024))) uint16_t lds[2][2][WSE];
    __shared__ float rv_s[LB];
    __shared__ float2 zs[ZR && !IS_DW ? LB : 1];
    wide_tile<IS_DW ? kWideDW : kWideDH, TO, NW, ZR>(a, blockIdx.x, lds, rv_s, zs);
}

// The head forward Z = H W (+ b) in bf16 on the same tiles (fp32 accumulation, one rounding of Z); FS:
// with the per-tile row statistics in the epilogue (a kernel of its own: the statistics epilogue's
// registers would otherwise constrain the plain forward's k loop).
template <typename TO, int NW, bool FS = false>
__global__ __launch_bounds__(NW * 64, 1) void lds256w_fwd_kernel(WideArgs a) {
    __shared__ __attribute__((aligned(1024))) uint16_t lds[2][2][WSE];
    __shared__ float rv_s[LB];
    wide_tile<kWideFWD, TO, NW, false, FS>(a, blockIdx.x, lds, rv_s);
}

// Both products in one grid: blocks [0, nh) run dH's units (the long k ranges first), the rest dW's
// tiles, so that the shorter dW tiles fill the compute units that dH's last round leaves idle instead of
// a second launch starting after a partly empty round. nh is a multiple of 8, so each part keeps its
// own XCD order.
template <typename TO, int NW, bool ZR = false>
__global__ __launch_bounds__(NW * 64, 1) void lds256w_pair_kernel(WideArgs h, WideArgs w, int nh) {
    __shared__ __attribute__((aligned(1024))) uint16_t lds[2][2][WSE];
    __shared__ float rv_s[LB];
    __shared__ float2 zs[ZR ? LB : 1];
    if ((int)blockIdx.x < nh) wide_tile<kWideDH, TO, NW, ZR>(h, blockIdx.x, lds, rv_s, zs);
    else wide_tile<kWideDW, float, NW, ZR>(w, (int)blockIdx.x - nh, lds, rv_s);
}

// Split-K reduction for the rank-1 form over the rectangle [pm0, M) x [pn0, Nn) of the output, in split
// order: out = sum_z part[z] + rv[m] cv[n] (+ beta out); part[z] is that rectangle, row-major.
template <typename TO>
__global__ __launch_bounds__(256) void splitk_rank1_kernel(const float* __restrict__ part, int splits, int M, int Nn,
                                                           int pm0, int pn0, const float* __restrict__ rv,
                                                           const float* __restrict__ cv, TO* __restrict__ out,
                                                           int64_t ldo, float beta) {
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t Nr = Nn - pn0;
    const int64_t MN = (int64_t)(M - pm0) * Nr;
    if (idx >= MN) return;
    const int64_t m = pm0 + idx / Nr, n = pn0 + idx % Nr;
    float a = 0.f;
    for (int z = 0; z < splits; ++z) a += part[(int64_t)z * MN + idx];
    if (rv != nullptr) a = fmaf(rv[m], cv[n], a);
    if (beta != 0.f) a += beta * ldf<TO>(out, m * ldo + n);
    stf<TO>(out, m * ldo + n, a);
}

// Rank-1 vectors. Blocks [0, nu): chunk sums of W q_hat, one wave per (row n of W, chunk c of ucw columns),
// four 16-byte loads of W (and the matching q_hat) in flight per lane: upart[c][n]. Blocks
// [nu, ...): partial column sums of H over rows in I, kHsRows rows by 512 columns per block (wave w adds rows
// w, w + 4, ...; the four wave sums are added in wave order).
constexpr int kHsRows = 128;
__global__ __launch_bounds__(256) void vjp_rank1_kernel(const uint16_t* __restrict__ W, int64_t ldw, int d, int V,
                                                        const float* __restrict__ q_hat, int nu, int uch, int ucw,
                                                        const uint16_t* __restrict__ H, int64_t ldh, int N,
                                                        const int32_t* __restrict__ labels, int32_t ignore_index,
                                                        float* __restrict__ upart, float* __restrict__ hpart) {
    const int l = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    if ((int)blockIdx.x < nu) {
        // nu * 4 (at most kUWaves) waves take the d * uch units in turn
        for (int unit = blockIdx.x * 4 + wave; unit < d * uch; unit += nu * 4) {
            const int n = unit / uch, c = unit % uch;
            const uint16_t* wr = W + (int64_t)n * ldw;
            const int j1 = min(V, (c + 1) * ucw);   // V and the chunk bounds are multiples of 8
            float acc[4] = {0.f, 0.f, 0.f, 0.f};
            for (int j = c * ucw + l * 8; j < j1; j += 4 * 512) {
                uint4 w[4];
                float4 q[8];
                // all loads unconditional (clamped to the chunk's last 8 columns, which exist) so that they are in
                // flight together; the W of a clamped load is masked to zero
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const int jj = min(j + k * 512, j1 - 8);
                    w[k] = *reinterpret_cast<const uint4*>(wr + jj);
                    q[2 * k] = *reinterpret_cast<const float4*>(q_hat + jj);
                    q[2 * k + 1] = *reinterpret_cast<const float4*>(q_hat + jj + 4);
                }
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const uint32_t mk = lane_mask(j + k * 512 < j1);
                    w[k] = make_uint4(w[k].x & mk, w[k].y & mk, w[k].z & mk, w[k].w & mk);
                }
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    acc[k] += bf16_lo(w[k].x) * q[2 * k].x + bf16_hi(w[k].x) * q[2 * k].y + bf16_lo(w[k].y) * q[2 * k].z +
                              bf16_hi(w[k].y) * q[2 * k].w + bf16_lo(w[k].z) * q[2 * k + 1].x + bf16_hi(w[k].z) * q[2 * k + 1].y +
                              bf16_lo(w[k].w) * q[2 * k + 1].z + bf16_hi(w[k].w) * q[2 * k + 1].w;
            }
            const float sum = wave_sum((acc[0] + acc[1]) + (acc[2] + acc[3]));
            if (l == 0) upart[(int64_t)c * d + n] = sum;
        }
        return;
    }
    __shared__ float sh[4][512];
    const int b = blockIdx.x - nu;
    const int ncb = (d + 511) / 512;
    const int cb = b % ncb, rb = b / ncb;
    const int col = cb * 512 + l * 8;
    const int colc = col < d ? col : d - 8;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    const int rbeg = rb * kHsRows;
    // rows rbeg + wave + 4e, e < kHsRows / 4: all loads of a group of 8 rows in flight together
#pragma unroll
    for (int e0 = 0; e0 < kHsRows / 4; e0 += 8) {
        uint4 h[8];
        float mk[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int i = rbeg + wave + 4 * (e0 + e);
            const int ic = i < N ? i : N - 1;
            // the label is loaded unconditionally (ic is clamped) and tested without short-circuit evaluation,
            // so that no load moves under a branch and all of the group's loads are in flight together
            const int32_t lab = labels[ic];
            const bool ok = (i < N) & (lab != ignore_index) & (lab >= 0) & ((int64_t)lab < V);
            mk[e] = ok ? 1.f : 0.f;
            h[e] = *reinterpret_cast<const uint4*>(H + (int64_t)ic * ldh + colc);
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            acc[0] += mk[e] * bf16_lo(h[e].x);
            acc[1] += mk[e] * bf16_hi(h[e].x);
            acc[2] += mk[e] * bf16_lo(h[e].y);
            acc[3] += mk[e] * bf16_hi(h[e].y);
            acc[4] += mk[e] * bf16_lo(h[e].z);
            acc[5] += mk[e] * bf16_hi(h[e].z);
            acc[6] += mk[e] * bf16_lo(h[e].w);
            acc[7] += mk[e] * bf16_hi(h[e].w);
        }
    }
#pragma unroll
    for (int c = 0; c < 8; ++c) sh[wave][l * 8 + c] = acc[c];
    __syncthreads();
    for (int c = threadIdx.x; c < 512; c += 256) {
        const int m = cb * 512 + c;
        if (m < d) hpart[(int64_t)rb * d + m] = ((sh[0][c] + sh[1][c]) + sh[2][c]) + sh[3][c];
    }
}


// Split-K reduction in split order: out = sum_z part[z] (+ beta * out for dW).
template <typename TO>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part, int splits, int M, int Nn,
                                                            TO* __restrict__ out, int64_t ldo, float beta) {
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t MN = (int64_t)M * Nn;
    if (idx >= MN) return;
    float a = 0.f;
    for (int z = 0; z < splits; ++z) a += part[(int64_t)z * MN + idx];
    const int64_t m = idx / Nn, n = idx % Nn;
    if (beta != 0.f) a += beta * ldf<TO>(out, m * ldo + n);
    stf<TO>(out, m * ldo + n, a);
}

// ---- planning ------------------------------------------------------------------------------------
// ---- fused small products --------------------------------------------------------------------
// Both products of a small head in one launch, each in its rank-1 form, with nothing staged
// beforehand: workgroups [0, tw) own 64 x 64 tiles of dW = alpha H^T R + hsum cq^T, the rest
// 64 x 64 tiles of dH = alpha R W^T + mask u^T (alpha = (1 - lambda)/N_t, cq = lambda q_hat/N_t,
// hsum_m = sum over rows in I of H[k][m], u = W cq). Each workgroup runs over the whole k range
// (no split-K, no partial sums): k tiles of 64 go through two LDS buffers, with four tiles in flight
// in registers. The rank-1 vectors a tile needs come from the same copies on their way to LDS:
// a dW tile sums its H columns over the rows in I, a dH tile dots its W rows with q_hat. dW's
// operands are k-major in memory (rows k of H and R) and reach the MFMA through transposing LDS
// reads; dH's are k-contiguous and use 16-byte reads. The dW tiles of the first row of tiles also
// write db.
constexpr int FB = 64;     // output tile
constexpr int FK = 64;     // k tile
constexpr int FSETS = 4;   // k tiles in flight in registers

struct FusedArgs {
    const uint16_t* H; int64_t ldh;
    const uint16_t* W; int64_t ldw;
    const uint16_t* R; int64_t ldr;
    const int32_t* labels; int32_t ig;
    const float* q_hat; const float* s; const int32_t* n_valid; float lambda;
    int N, d, V;
    float* dW; int64_t lddw; float beta;
    void* dH; int64_t lddh; int dh_bf16;
    float* db;
    int tw_n, tw, th_n;   // dW tiles along V, dW tile count, dH tiles along d
    const float* row_lse; // logits input: R is formed from Z (the R argument) and lse; null: R is stored
};

// element offset of (row, col) in a 64 x 64 bf16 LDS tile whose 16-byte chunks are swizzled by row
__device__ __forceinline__ int ftile_off(int row, int col) { return row * FB + ((((col >> 3) ^ (row & 7))) << 3) + (col & 7); }

template <bool is_dw>
__device__ __forceinline__ void fused_tile(const FusedArgs& a, int id, uint16_t (&sa)[2][FK * FB],
                                           uint16_t (&sb)[2][FK * FB], float (&red)[FB][33], float (&vec)[FB]) {
    const int t = threadIdx.x, l = t % kWave;
    const int wave = __builtin_amdgcn_readfirstlane(t / kWave);
    const int wm = wave / 2, wn = wave % 2;
    const int m0 = (id / (is_dw ? a.tw_n : a.th_n)) * FB, n0 = (id % (is_dw ? a.tw_n : a.th_n)) * FB;
    const int M = is_dw ? a.d : a.N, Nn = is_dw ? a.V : a.d, K = is_dw ? a.N : a.V;
    const int nt = *a.n_valid;
    const float alpha = nt > 0 ? (float)((1.0 - (double)a.lambda) / (double)nt) : 0.f;
    const double cscale = nt > 0 ? (double)a.lambda / (double)nt : 0.0;
    const int nk = ((K + FK - 1) / FK + FSETS - 1) / FSETS * FSETS;   // tiles past K hold zeros

    // copy geometry: chunks t and t + 256 of each operand's 64 x 64 tile: tile row t/8 + 32 e,
    // 16-byte chunk lc = t % 8 of that row
    const int lc = t % 8;
    const int r0 = t / 8;
    // operand A: dW -> H rows k, columns m0 + 8 lc; dH -> R rows m0 + r, k chunk 8 lc
    // operand B: dW -> R rows k, columns n0 + 8 lc; dH -> W rows n0 + r, k chunk 8 lc
    const uint16_t* pa = is_dw ? a.H : a.R;
    const uint16_t* pb = is_dw ? a.R : a.W;
    const int64_t lda = is_dw ? a.ldh : a.ldr, ldb = is_dw ? a.ldr : a.ldw;
    const int rows_a = is_dw ? a.N : a.N, rows_b = is_dw ? a.N : a.d;
    const auto da = make_desc(pa, (int)(((int64_t)(rows_a - 1) * lda + (is_dw ? a.d : a.V)) * 2));
    const auto db_ = make_desc(pb, (int)(((int64_t)(rows_b - 1) * ldb + a.V) * 2));
    auto off_a = [&](int k0, int e) {
        const int r = r0 + 32 * e;
        if constexpr (is_dw) {
            const int k = k0 + r, m = m0 + lc * 8;
            return (k < a.N && m < a.d) ? (int)(((int64_t)k * lda + m) * 2) : kOob;
        }
        const int i = m0 + r, k = k0 + lc * 8;
        return (i < a.N && k < a.V) ? (int)(((int64_t)i * lda + k) * 2) : kOob;
    };
    auto off_b = [&](int k0, int e) {
        const int r = r0 + 32 * e;
        if constexpr (is_dw) {
            const int k = k0 + r, n = n0 + lc * 8;
            return (k < a.N && n < a.V) ? (int)(((int64_t)k * ldb + n) * 2) : kOob;
        }
        const int j = n0 + r, k = k0 + lc * 8;
        return (j < a.d && k < a.V) ? (int)(((int64_t)j * ldb + k) * 2) : kOob;
    };
    // one k tile in registers: the four 16-byte copies and what the rank-1 sums need with them
    struct Set {
        u32x4_t c[4];
        int lab[2];     // dW: labels of the two H rows (rows past N: ignore_index)
        float4 q[2];    // dH: q_hat over the chunk's 8 k
        float zl[2];    // dW with logits input: lse of the two R rows
        int kt;
    };
    const bool zin = a.row_lse != nullptr;
    // dH with logits input: c and label of this thread's two R rows (fixed over k)
    float zc_h[2] = {INFINITY, INFINITY};
    int zy_h[2] = {-1, -1};
    if (!is_dw && zin) {
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const int i = m0 + r0 + 32 * e;
            if (i < a.N) {
                zc_h[e] = z_row_c(a.row_lse, a.labels, i, a.V, a.ig);
                zy_h[e] = a.labels[i];
            }
        }
    }
    auto load_set = [&](Set& st, int kt) {
        const int k0 = kt * FK;
        st.kt = kt;
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            st.c[e] = __builtin_amdgcn_raw_buffer_load_b128(da, off_a(k0, e), 0, 0);
            st.c[2 + e] = __builtin_amdgcn_raw_buffer_load_b128(db_, off_b(k0, e), 0, 0);
        }
        if constexpr (is_dw) {
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                const int k = k0 + r0 + 32 * e;
                st.lab[e] = a.labels[k < a.N ? k : a.N - 1];
                if (zin) st.zl[e] = a.row_lse[k < a.N ? k : a.N - 1];
                if (k >= a.N) st.lab[e] = a.ig;
            }
        } else {
            const int k = k0 + lc * 8;
            const int kc = k < a.V ? k : a.V - 8;
            st.q[0] = *reinterpret_cast<const float4*>(a.q_hat + kc);
            st.q[1] = *reinterpret_cast<const float4*>(a.q_hat + kc + 4);
            if (k >= a.V) st.q[0] = st.q[1] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
    };
    float part[8];   // dW: sums of this thread's 8 H columns over rows in I; dH: [0..1] dots of its 2 W rows
#pragma unroll
    for (int e = 0; e < 8; ++e) part[e] = 0.f;
    auto write_set = [&](const Set& st, int buf) {
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const int r = r0 + 32 * e;
            const int o = r * FB + ((lc ^ (r & 7)) << 3);
            u32x4_t ca = st.c[e], cb = st.c[2 + e];
            if (zin) {
                if constexpr (is_dw) {   // R is operand B: row k0 + r, columns n0 + 8 lc
                    bool bad = false;
                    const bool valid = label_valid(st.lab[e], a.V, a.ig, &bad);
                    const int n = n0 + lc * 8;
                    cb = z_chunk_to_r(cb, valid ? st.zl[e] * kLog2e : INFINITY, st.lab[e] - n, n < a.V);
                } else {                 // R is operand A: row m0 + r, k chunk kt FK + 8 lc
                    const int k = st.kt * FK + lc * 8;
                    ca = z_chunk_to_r(ca, zc_h[e], zy_h[e] - k, k < a.V);
                }
            }
            *reinterpret_cast<u32x4_t*>(&sa[buf][o]) = ca;
            *reinterpret_cast<u32x4_t*>(&sb[buf][o]) = cb;
        }
        if constexpr (is_dw) {
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                bool bad = false;
                const float vm = label_valid(st.lab[e], a.V, a.ig, &bad) ? 1.f : 0.f;
#pragma unroll
                for (int p = 0; p < 4; ++p) {
                    part[2 * p] = fmaf(vm, bf16_lo(st.c[e][p]), part[2 * p]);
                    part[2 * p + 1] = fmaf(vm, bf16_hi(st.c[e][p]), part[2 * p + 1]);
                }
            }
        } else {
            const float q8[8] = {st.q[0].x, st.q[0].y, st.q[0].z, st.q[0].w, st.q[1].x, st.q[1].y, st.q[1].z, st.q[1].w};
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                float acc = part[e];
#pragma unroll
                for (int p = 0; p < 4; ++p) {
                    acc = fmaf(bf16_lo(st.c[2 + e][p]), q8[2 * p], acc);
                    acc = fmaf(bf16_hi(st.c[2 + e][p]), q8[2 * p + 1], acc);
                }
                part[e] = acc;
            }
        }
    };
    // fragments of MFMA step s (k = 16 s .. 16 s + 15) of the tile in buffer buf
    auto read_frags = [&](int buf, int s, bf16x8_t& fa, bf16x8_t& fb) {
        if constexpr (is_dw) {
            const int g = l / 16, sl = l % 16;
            const int kr = 16 * s + (g / 2) * 8 + sl / 4;
            const int ca = wm * 32 + (g % 2) * 16 + (sl % 4) * 4, cb = wn * 32 + (g % 2) * 16 + (sl % 4) * 4;
            const v4s_t a0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t*)&sa[buf][ftile_off(kr, ca)]);
            const v4s_t a1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t*)&sa[buf][ftile_off(kr + 4, ca)]);
            const v4s_t b0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t*)&sb[buf][ftile_off(kr, cb)]);
            const v4s_t b1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t*)&sb[buf][ftile_off(kr + 4, cb)]);
            fa = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7));
            fb = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(b0, b1, 0, 1, 2, 3, 4, 5, 6, 7));
        } else {
            const int ra = wm * 32 + l % 32, rb = wn * 32 + l % 32, c = 2 * s + l / 32;
            fa = *reinterpret_cast<const bf16x8_t*>(&sa[buf][ra * FB + ((c ^ (ra & 7)) << 3)]);
            fb = *reinterpret_cast<const bf16x8_t*>(&sb[buf][rb * FB + ((c ^ (rb & 7)) << 3)]);
        }
    };

    f32x16_t acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
    Set sets[FSETS];
#pragma unroll
    for (int q = 0; q < FSETS; ++q) load_set(sets[q], q);
    write_set(sets[0], 0);
    load_set(sets[0], FSETS);
    __syncthreads();
    // iteration kt: read tile kt (buffer kt % 2), write tile kt + 1 into the other buffer from its
    // register set and reload that set with tile kt + 1 + FSETS, then the four MFMA steps
    for (int kt0 = 0; kt0 < nk; kt0 += FSETS) {
#pragma unroll
        for (int u = 0; u < FSETS; ++u) {
            const int kt = kt0 + u;
            const int buf = u & 1;
            bf16x8_t fa[4], fb[4];
#pragma unroll
            for (int s = 0; s < 4; ++s) read_frags(buf, s, fa[s], fb[s]);
            Set& st = sets[(u + 1) % FSETS];
            write_set(st, buf ^ 1);
            load_set(st, kt + 1 + FSETS);
#pragma unroll
            for (int s = 0; s < 4; ++s) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[s], fb[s], acc, 0, 0, 0);
            __syncthreads();
        }
    }

    // rank-1 vectors of the tile: dW -> hsum over its 64 columns, dH -> u over its 64 rows of W
    if (is_dw) {
#pragma unroll
        for (int e = 0; e < 8; ++e) red[lc * 8 + e][r0] = part[e];
    } else {
        red[r0][lc] = part[0];
        red[r0 + 32][lc] = part[1];
    }
    __syncthreads();
    if (t < FB) {
        float v = 0.f;
        const int nc = is_dw ? 32 : 8;
        for (int c = 0; c < nc; ++c) v += red[t][c];
        vec[t] = is_dw ? v : (float)(cscale * (double)v);
    }
    __syncthreads();
    // accumulator element r of lane l: tile row wm*32 + (r/4)*8 + (l/32)*4 + r%4, column wn*32 + l%32
    const int col = wn * 32 + l % 32;
    const int n = n0 + col;
    float cqn = 0.f;
    if (is_dw && n < Nn) cqn = (float)(cscale * (double)a.q_hat[n]);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int row = wm * 32 + (r / 4) * 8 + (l / 32) * 4 + r % 4;
        const int m = m0 + row;
        if (m >= M || n >= Nn) continue;
        if (is_dw) {
            float x = fmaf(alpha, acc[r], vec[row] * cqn);
            float* p = a.dW + (int64_t)m * a.lddw + n;
            *p = a.beta != 0.f ? x + a.beta * *p : x;
        } else {
            bool bad = false;
            const float vm = label_valid(a.labels[m], a.V, a.ig, &bad) ? 1.f : 0.f;
            const float x = fmaf(alpha, acc[r], vm * vec[col]);
            if (a.dh_bf16) stf<uint16_t>(static_cast<uint16_t*>(a.dH), (int64_t)m * a.lddh + n, x);
            else stf<float>(static_cast<float*>(a.dH), (int64_t)m * a.lddh + n, x);
        }
    }
    if (is_dw && m0 == 0 && a.db != nullptr && t < FB && n0 + t < a.V) {
        const int j = n0 + t;
        a.db[j] = nt > 0 ? (1.0f - a.lambda) * a.s[j] + a.lambda * a.q_hat[j] : 0.f;
    }
}

__global__ __launch_bounds__(256, 2) void vjp_fused_small_kernel(FusedArgs a) {
    __shared__ __attribute__((aligned(16))) uint16_t sa[2][FK * FB];
    __shared__ __attribute__((aligned(16))) uint16_t sb[2][FK * FB];
    __shared__ float red[FB][33];
    __shared__ float vec[FB];
    if ((int)blockIdx.x < a.tw) fused_tile<true>(a, (int)blockIdx.x, sa, sb, red, vec);
    else fused_tile<false>(a, (int)blockIdx.x - a.tw, sa, sb, red, vec);
}

constexpr int kCUs = 256;        // MI355X compute units
constexpr int kMaxSplits = 8;

// kRank1: the 256-tile rank-1 form on the 64-deep kernel (lds256w_kernel)
enum GemmKind { kSimt = 0, kMfma128 = 1, kRank1 = 4 };
struct GemmPlan {
    int kind, splits;
    // rank-1 kind: outer tiles [0, outer_dp) run with the whole k range, the rest with `splits`
    int outer_dp = 0;
};
struct Plan {
    GemmPlan w, h;
    // both 64-deep products in one grid (dH's units first, then dW's tiles): h.splits is dH's k split,
    // dW runs unsplit
    bool pair = false;
};

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Split-K factor: modelled time = rounds of resident workgroups x per-tile k work, plus the
// partial-sum traffic (write and read of fp32 partials) at streaming bandwidth.
int choose_splits(int64_t tiles, int64_t M, int64_t N, int64_t K, int tb, int ktile, int per_cu) {
    const double tile_flop_rate = 2.0 * 2.5e15 / kCUs / per_cu / 2;  // ~half of the per-workgroup MFMA share
    int best = 1;
    double best_t = 1e300;
    for (int s = 1; s <= kMaxSplits; ++s) {
        const int64_t kps = cdiv(cdiv(K, s), ktile) * ktile;
        if (s > 1 && kps < 4LL * ktile) break;
        const int64_t units = tiles * s;
        const int64_t rounds = cdiv(units, (int64_t)kCUs * per_cu);
        double t = rounds * (2.0 * tb * tb * kps) / tile_flop_rate;
        if (s > 1) t += (2.0 * s + 1.0) * 4.0 * M * N / 5e12;
        if (t < best_t * 0.98) {
            best_t = t;
            best = s;
        }
    }
    return best;
}

// Schedule of the 64-deep 256-tile kernel. Each XCD (32 CUs) runs the inner tiles of the (outer
// tile, k split) pairs dealt to it, 32 workgroups at a time. Whole rounds of outer tiles run over the
// full k range; the outer tiles left over (a partly filled last round) split k into `splits` parts so
// that their pairs spread over all XCDs, and a reduction pass sums their fp32 partials in split order.
// Modelled time: rounds per XCD x k tiles per split x the measured time of one 256 x 256 x 64 tile
// step, plus the partial-sum traffic (write, read, and the output) at streaming bandwidth.
GemmPlan plan_wide(int64_t M, int64_t N, int64_t K, bool inner_is_m) {
    constexpr double kTileStep = 1.8e-6;   // seconds per 256 x 256 x 64 tile step
    constexpr int64_t kXcd = 8, kCuPerXcd = kCUs / 8;
    const int64_t MT = cdiv(M, LB), NT = cdiv(N, LB);
    const int64_t inner = inner_is_m ? MT : NT, outer = inner_is_m ? NT : MT;
    const int64_t nk = cdiv(K, WKT);
    auto rounds = [&](int64_t pairs) { return cdiv(cdiv(pairs, kXcd) * inner, kCuPerXcd); };
    const int64_t per_round = kXcd * std::max<int64_t>(1, kCuPerXcd / inner);   // outer tiles per whole round
    const int64_t full = (outer / per_round) * per_round;
    GemmPlan best{kRank1, 1};
    best.outer_dp = (int)outer;
    double best_t = (double)rounds(outer) * nk * kTileStep;
    for (int64_t dp : {(int64_t)0, full}) {
        const int64_t rem = outer - dp;
        if (rem <= 0) continue;
        const int64_t rect = inner_is_m ? M * std::max<int64_t>(0, N - dp * LB) : std::max<int64_t>(0, M - dp * LB) * N;
        const double t_dp = (double)rounds(dp) * nk * kTileStep;
        for (int s = 1; s <= 16; ++s) {
            const int64_t kps = cdiv(nk, s);
            if (s > 1 && kps < 4) break;
            double t = t_dp + (double)rounds(rem * s) * kps * kTileStep;
            if (s > 1) t += (2.0 * s + 2.0) * 4.0 * (double)rect / 5e12;
            if (t < best_t - 2e-6) {   // a gain of at least 2 us
                best_t = t;
                best.splits = s;
                best.outer_dp = (int)dp;
            }
        }
    }
    return best;
}

GemmPlan plan_gemm(bool mfma, bool big_ok, int64_t M, int64_t N, int64_t K, bool inner_is_m) {
    if (!mfma || !big_ok) return {kSimt, choose_splits(cdiv(M, SB) * cdiv(N, SB), M, N, K, SB, SK, 4)};
    // large products: 256-tile rank-1 kernel; small ones (a few dozen 256 tiles or a short k) are
    // latency bound and run faster on the 128-tile kernel, which needs no rank-1 pre-pass
    const int64_t t256 = cdiv(M, LB) * cdiv(N, LB);
    if (t256 >= 24 && K >= 4 * WKT) return plan_wide(M, N, K, inner_is_m);
    // 128 tiles: split k so that every workgroup loads its whole k range at once, when that takes
    // at most kMaxSplits splits
    const int64_t t128 = cdiv(M, MB) * cdiv(N, MB);
    const int64_t s_pre = cdiv(K, (int64_t)kPre * MK);
    if (s_pre <= kMaxSplits) return {kMfma128, (int)s_pre};
    return {kMfma128, choose_splits(t128, M, N, K, MB, MK, 2)};
}

// Plan override for A/B measurement (environment BOM_VJP_PLAN = "kind_w,splits_w,kind_h,splits_h",
// read once; 0 keeps the automatic choice (small products: the fused launch); kinds 1 = 128-tile
// MFMA (and no fused launch), 4 = 256-tile rank-1 kernel; splits > 0 force that k split on every tile).
struct PlanOverride {
    int kw = 0, sw = 0, kh = 0, sh = 0;
};
const PlanOverride& plan_override() {
    static const PlanOverride o = [] {
        PlanOverride r;
        if (const char* e = getenv("BOM_VJP_PLAN")) sscanf(e, "%d,%d,%d,%d", &r.kw, &r.sw, &r.kh, &r.sh);
        if (r.sw < 0 || r.sw > kMaxSplits) r.sw = 0;
        if (r.sh < 0 || r.sh > kMaxSplits) r.sh = 0;
        return r;
    }();
    return o;
}

// Waves per workgroup of the 64-deep kernels, per product (dH, dW, forward, the pair launch): four, or
// eight (two per SIMD). Environment BOM_VJP_WAVES = "dH,dW,fwd,pair" overrides for A/B measurement
// (read once; values other than 4 and 8 keep the default).
struct WaveCfg {
    int dh = 8, dw = 8, fwd = 8, pair = 8;
};
const WaveCfg& wave_cfg() {
    static const WaveCfg c = [] {
        WaveCfg r;
        int v[4] = {0, 0, 0, 0};
        if (const char* e = getenv("BOM_VJP_WAVES")) sscanf(e, "%d,%d,%d,%d", &v[0], &v[1], &v[2], &v[3]);
        int* f[4] = {&r.dh, &r.dw, &r.fwd, &r.pair};
        for (int i = 0; i < 4; ++i)
            if (v[i] == 4 || v[i] == 8) *f[i] = v[i];
        return r;
    }();
    return c;
}

// Blocked XCD order of whole-round launches (see unit_of) for more than 8 inner tiles (a multiple of 8):
// at the 8B shape a third fewer L2 misses on both VJP products (dH 37.8 -> 25.2 GB per launch) at the same
// time; the forward (inner tiles along N) runs 3-7 % faster with it at the 8B, 1B and 32K shapes.
// Environment BOM_VJP_XCD_BLOCK = 0 selects the plain order for A/B measurement (read once).
int xcd_blocked(int inner) {
    static const int mode = [] {
        const char* e = getenv("BOM_VJP_XCD_BLOCK");
        return e ? atoi(e) : 1;
    }();
    return (mode == 1 && inner > 8 && inner % 8 == 0) ? 1 : 0;
}

void apply_override(GemmPlan& g, int kind, int splits, int64_t M, int64_t N, int64_t K) {
    if (g.kind == kSimt) return;
    if (kind == kMfma128) {
        g.kind = kMfma128;
        g.outer_dp = 0;
    }
    if (kind == kRank1) g.kind = kRank1;

    if (splits > 0) {
        const int ktile = g.kind == kRank1 ? WKT : MK;
        // every split keeps at least one k tile
        g.splits = (int)(splits < cdiv(K, ktile) ? splits : cdiv(K, ktile));
        g.outer_dp = 0;   // a forced split applies to every tile
    }
    (void)M;
    (void)N;
}

// Completion time, in 256 x 256 x 64 tile steps, of one launch of the 64-deep kernel: parts in block
// order, each (pairs, inner tiles per pair, k tile steps per unit); pair q of a part goes to XCD q % 8
// and its inner tiles follow each other there; each XCD starts its blocks in order on the first of its
// 32 compute units to become free (greedy list schedule).
double sim_launch(std::initializer_list<std::array<int64_t, 3>> parts) {
    double end = 0.0;
    for (int x = 0; x < 8; ++x) {
        std::priority_queue<double, std::vector<double>, std::greater<double>> cu;
        for (int c = 0; c < kCUs / 8; ++c) cu.push(0.0);
        for (const auto& pt : parts)
            for (int64_t q = x; q < pt[0]; q += 8)
                for (int64_t i = 0; i < pt[1]; ++i) {
                    const double t = cu.top() + (double)pt[2];
                    cu.pop();
                    cu.push(t);
                }
        while (cu.size() > 1) cu.pop();
        end = std::max(end, cu.top());
    }
    return end;
}

// Whether one grid with both products (dH first) beats the two launches of the separate plans, and with
// which k split of dH. Times in tile steps; split partials cost their fp32 write, read and the output.
void plan_pair(Plan& p, int64_t N, int64_t d, int64_t V) {
    constexpr double kStep = 1.8e-6, kBw = 5e12;
    const int64_t inner = cdiv(d, LB);
    const int64_t ow = cdiv(V, LB), oh = cdiv(N, LB);
    const int64_t nkw = cdiv(N, WKT), nkh = cdiv(V, WKT);
    auto red = [&](int s, int64_t rect) { return s > 1 ? (2.0 * s + 2.0) * 4.0 * (double)rect / kBw / kStep : 0.0; };
    // separate launches as planned (each split launch followed by its reduction)
    auto sep = [&](const GemmPlan& g, int64_t outer, int64_t nk, int64_t rect_per_outer) {
        const int64_t dp = std::min<int64_t>(g.outer_dp, outer);
        double t = dp > 0 ? sim_launch({{dp, inner, nk}}) : 0.0;
        if (dp < outer) {
            t += sim_launch({{(outer - dp) * g.splits, inner, cdiv(nk, g.splits)}});
            t += red(g.splits, (outer - dp) * rect_per_outer);
        }
        return t;
    };
    const double t_sep = sep(p.w, ow, nkw, LB * d) + sep(p.h, oh, nkh, LB * d);
    double best = t_sep * 0.95;
    int best_s = 0;
    for (int s = 1; s <= 16; ++s) {
        if (s > 1 && cdiv(nkh, s) < 4) break;
        const double t = sim_launch({{oh * s, inner, cdiv(nkh, s)}, {ow, inner, nkw}}) + red(s, N * d);
        if (t < best) {
            best = t;
            best_s = s;
        }
    }
    if (best_s == 0) return;
    p.pair = true;
    p.h.splits = best_s;
    p.h.outer_dp = 0;
    p.w.splits = 1;
    p.w.outer_dp = (int)ow;
}

Plan make_plan_uncached(int64_t N, int64_t d, int64_t V, bom_dtype dt) {
    const bool mfma = dt == BOM_BF16;
    Plan p;
    // the MFMA kernels load whole 16-byte chunks: extents along k and along contiguous rows must be
    // multiples of 8 (H^T rows have N elements); other shapes use the SIMT kernels
    const bool m8 = N % 8 == 0 && d % 8 == 0 && V % 8 == 0;
    p.w = plan_gemm(mfma, m8, d, V, N, true);    // dW: M = d, N = V, K = rows; inner tiles along d
    p.h = plan_gemm(mfma, m8, N, d, V, false);   // dH: M = rows, N = d, K = V
    const PlanOverride& o = plan_override();
    apply_override(p.w, o.kw, o.sw, d, V, N);
    apply_override(p.h, o.kh, o.sh, N, d, V);
    if (o.kw == 0 && o.kh == 0 && o.sw == 0 && o.sh == 0 && p.w.kind == kRank1 && p.h.kind == kRank1)
        plan_pair(p, N, d, V);
    return p;
}

// Plans are deterministic functions of the shape; the schedule simulation is kept per shape.
Plan make_plan(int64_t N, int64_t d, int64_t V, bom_dtype dt) {
    static std::mutex mu;
    static std::map<std::array<int64_t, 4>, Plan> cache;
    const std::array<int64_t, 4> key{N, d, V, (int64_t)dt};
    {
        std::lock_guard<std::mutex> lk(mu);
        auto it = cache.find(key);
        if (it != cache.end()) return it->second;
    }
    const Plan p = make_plan_uncached(N, d, V, dt);
    std::lock_guard<std::mutex> lk(mu);
    if (cache.size() < 256) cache.emplace(key, p);
    return p;
}

// Plan of the SIMT kernels, which run bf16 operands that the MFMA kernels cannot stage (a leading
// dimension that is not a multiple of 8, or a base that is not 16-byte aligned): SIMT tiles with their own
// k split over every tile.
Plan simt_plan(int64_t N, int64_t d, int64_t V) {
    Plan p;
    p.w = plan_gemm(false, false, d, V, N, true);
    p.h = plan_gemm(false, false, N, d, V, false);
    return p;
}

// Bytes of fp32 split-K partials a plan writes: the rectangle of the tiles that split k (all of them
// unless the wide kernel runs outer tiles [0, outer_dp) unsplit); dW and dH share the buffer.
size_t partial_bytes(const Plan& p, int64_t N, int64_t d, int64_t V) {
    const int64_t wcols = std::max<int64_t>(0, V - (int64_t)p.w.outer_dp * LB);
    const int64_t hrows = std::max<int64_t>(0, N - (int64_t)p.h.outer_dp * LB);
    const bool ww = p.w.kind == kRank1, hw = p.h.kind == kRank1;
    const size_t pw = p.w.splits > 1 ? (size_t)p.w.splits * d * (ww ? wcols : V) * 4 : 0;
    const size_t ph = p.h.splits > 1 ? (size_t)p.h.splits * (hw ? hrows : N) * d * 4 : 0;
    return std::max(pw, ph);
}

VjpWs vjp_ws(int64_t N, int64_t d, int64_t V, bom_dtype dt) {
    const Plan p = make_plan(N, d, V, dt);
    VjpWs w;
    w.cq_off = 0;
    w.cqp_off = align256((size_t)V * 4);
    w.vmask_off = align256(w.cqp_off + (size_t)V * 4);
    w.scal_off = align256(w.vmask_off + (size_t)N * 4);
    const bool r1 = p.w.kind == kRank1 || p.h.kind == kRank1;
    w.zc_off = align256(w.scal_off + 16);
    w.hpart_off = align256(w.zc_off + (size_t)N * 4);
    w.hsum_off = align256(w.hpart_off + (r1 ? (size_t)cdiv(N, kHsRows) * d * 4 : 0));
    w.u_off = align256(w.hsum_off + (r1 ? (size_t)d * 4 : 0));
    w.upart_off = align256(w.u_off + (r1 ? (size_t)d * 4 : 0));
    w.part_off = align256(w.upart_off + (r1 ? (size_t)u_chunks(d, V) * d * 4 : 0));
    size_t need = partial_bytes(p, N, d, V);
    // the same call may take the SIMT plan (misaligned operands)
    if (dt == BOM_BF16) need = std::max(need, partial_bytes(simt_plan(N, d, V), N, d, V));
    w.total = align256(w.part_off + need);
    return w;
}

template <typename TO>
hipError_t run_gemm(bool is_dw, const GemmPlan& g, const void* A, int64_t lda, const void* B, int64_t ldb, bom_dtype dt,
                    int M, int Nn, int K, const Fold& f, TO* out, int64_t ldo, float beta, float* part, const float* rv,
                    const float* cv, hipStream_t st) {
    const int splits = g.splits;
    if (g.kind == kRank1) {
        // rank-1 form: out = alpha A B + rv cv^T (+ beta out)
        const int kt = WKT;
        const int kps = (int)(cdiv(cdiv(K, splits), kt) * kt);
        const int MT = (int)cdiv(M, LB), NT = (int)cdiv(Nn, LB);
        const int inner = is_dw ? MT : NT, outer = is_dw ? NT : MT;
        float* pz = splits > 1 ? part : nullptr;
        const uint16_t* a16 = static_cast<const uint16_t*>(A);
        const uint16_t* b16 = static_cast<const uint16_t*>(B);
        {
            // whole rounds over the full k range, then the leftover outer tiles with split k
            const int dp = std::min(g.outer_dp, outer);
            auto launch = [&](int ob, int oe, int nsplit, int kp, float* pp, const TileRange& tr) {
                dim3 gr((unsigned)(cdiv((int64_t)(oe - ob) * nsplit, 8) * 8 * inner));
                const WideArgs wa{a16, lda, b16, ldb, M, Nn, K, kp, tr, f.scal, rv, cv, out, ldo, beta, pp, nullptr,
                                  f.zc, f.labels};
                const int nw = is_dw ? wave_cfg().dw : wave_cfg().dh;
                if (f.zc != nullptr && is_dw)   // logits input: eight waves
                    hipLaunchKernelGGL((lds256w_kernel<true, float, 8, true>), gr, dim3(512), 0, st, wa);
                else if (f.zc != nullptr)
                    hipLaunchKernelGGL((lds256w_kernel<false, TO, 8, true>), gr, dim3(512), 0, st, wa);
                else if (is_dw && nw == 8)
                    hipLaunchKernelGGL((lds256w_kernel<true, float, 8>), gr, dim3(512), 0, st, wa);
                else if (is_dw)
                    hipLaunchKernelGGL((lds256w_kernel<true, float, 4>), gr, dim3(256), 0, st, wa);
                else if (nw == 8)
                    hipLaunchKernelGGL((lds256w_kernel<false, TO, 8>), gr, dim3(512), 0, st, wa);
                else
                    hipLaunchKernelGGL((lds256w_kernel<false, TO, 4>), gr, dim3(256), 0, st, wa);
                return hipGetLastError();
            };
            if (dp > 0) {
                const TileRange tr{inner, 0, dp, 1, 0, 0, 0, 0, xcd_blocked(inner)};
                hipError_t e = launch(0, dp, 1, (int)(cdiv(K, kt) * kt), nullptr, tr);
                if (e != hipSuccess) return e;
            }
            if (dp >= outer) return hipSuccess;
            const int pm0 = is_dw ? 0 : dp * LB, pn0 = is_dw ? dp * LB : 0;
            const int64_t ldp = Nn - pn0;
            const TileRange tr{inner, dp, outer, splits, pm0, pn0, ldp, (int64_t)(M - pm0) * ldp};
            hipError_t e = launch(dp, outer, splits, kps, pz, tr);
            if (e != hipSuccess || splits == 1) return e;
            const int64_t MN = (int64_t)(M - pm0) * ldp;
            hipLaunchKernelGGL(splitk_rank1_kernel<TO>, dim3((unsigned)cdiv(MN, 256)), dim3(256), 0, st, part, splits, M,
                               Nn, pm0, pn0, rv, cv, out, ldo, beta);
            return hipGetLastError();
        }
    }
    const int tb = g.kind == kMfma128 ? MB : SB;
    const int ktile = g.kind == kMfma128 ? MK : SK;
    int kps = (int)(cdiv(cdiv(K, splits), ktile) * ktile);
    float* pz = splits > 1 ? part : nullptr;
    const uint16_t* a16 = static_cast<const uint16_t*>(A);
    const uint16_t* b16 = static_cast<const uint16_t*>(B);
    {
        dim3 grid((unsigned)cdiv(Nn, tb), (unsigned)cdiv(M, tb), splits);
        if (g.kind == kMfma128) {
            if (is_dw)
                hipLaunchKernelGGL(mfma_dW_kernel, grid, dim3(256), 0, st, a16, lda, b16, ldb, M, Nn, K, kps, f,
                                   reinterpret_cast<float*>(out), ldo, beta, pz);
            else
                hipLaunchKernelGGL(mfma_dH_kernel<TO>, grid, dim3(256), 0, st, a16, lda, b16, ldb, M, Nn, K, kps, f, out,
                                   ldo, pz);
        } else if (dt == BOM_BF16) {
            if (is_dw)
                hipLaunchKernelGGL(simt_dW_kernel<uint16_t>, grid, dim3(256), 0, st, a16, lda, b16, ldb, M, Nn, K, kps, f,
                                   splits > 1 ? part : reinterpret_cast<float*>(out), ldo, beta, splits > 1 ? 0 : 1);
            else
                hipLaunchKernelGGL((simt_dH_kernel<uint16_t, TO>), grid, dim3(256), 0, st, a16, lda, b16, ldb, M, Nn, K,
                                   kps, f, out, ldo, part, splits > 1 ? 0 : 1);
        } else {
            const float* a32 = static_cast<const float*>(A);
            const float* b32 = static_cast<const float*>(B);
            if (is_dw)
                hipLaunchKernelGGL(simt_dW_kernel<float>, grid, dim3(256), 0, st, a32, lda, b32, ldb, M, Nn, K, kps, f,
                                   splits > 1 ? part : reinterpret_cast<float*>(out), ldo, beta, splits > 1 ? 0 : 1);
            else
                hipLaunchKernelGGL((simt_dH_kernel<float, TO>), grid, dim3(256), 0, st, a32, lda, b32, ldb, M, Nn, K, kps,
                                   f, out, ldo, part, splits > 1 ? 0 : 1);
        }
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || splits == 1) return e;
    const int64_t MN = (int64_t)M * Nn;
    hipLaunchKernelGGL(splitk_reduce_kernel<TO>, dim3((unsigned)cdiv(MN, 256)), dim3(256), 0, st, part, splits, M, Nn, out,
                       ldo, beta);
    return hipGetLastError();
}

}  // namespace

// bf16 dW / db (bf16 gradient storage): the products are formed in fp32 in the workspace past the
// products' own part, then rounded to nearest-even bf16 in one pass (dW = bf16(dW_fp32 + beta dW)).
size_t head_vjp_workspace_bytes(int64_t N, int64_t d, int64_t V, bom_dtype dt, bom_dtype dw_dt) {
    size_t n = vjp_ws(N, d, V, dt).total;
    if (dw_dt == BOM_BF16) n += align256((size_t)d * V * 4) + align256((size_t)V * 4);
    return n;
}

namespace {
__global__ __launch_bounds__(256) void round_dw_bf16_kernel(const float* __restrict__ src, int d, int V,
                                                            uint16_t* __restrict__ dW, int64_t lddw, float beta,
                                                            const float* __restrict__ db_src,
                                                            uint16_t* __restrict__ db) {
    const int64_t n = (int64_t)d * V;
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x; k < n + (db ? V : 0); k += stride) {
        if (k < n) {
            const int64_t i = k / V, j = k % V;
            uint16_t* p = dW + i * lddw + j;
            const float x = src[k];
            *p = f32_to_bf16(beta != 0.f ? x + beta * bf16_to_f32(*p) : x);
        } else {
            db[k - n] = f32_to_bf16(db_src[k - n]);
        }
    }
}
}  // namespace

hipError_t launch_head_vjp_f32(const HeadVjpArgs& a, hipStream_t st);

hipError_t launch_head_vjp(const HeadVjpArgs& a, hipStream_t st) {
    if (a.dw_dt != BOM_BF16) return launch_head_vjp_f32(a, st);
    HeadVjpArgs b = a;
    char* scratch = static_cast<char*>(a.ws) + vjp_ws(a.N, a.d, a.V, a.dt).total;
    b.dW = scratch;
    b.dw_dt = BOM_F32;
    b.lddw = a.V;
    b.dW_beta = 0.f;
    b.db = a.db ? scratch + align256((size_t)a.d * a.V * 4) : nullptr;
    hipError_t e = launch_head_vjp_f32(b, st);
    if (e != hipSuccess) return e;
    const int64_t n = (int64_t)a.d * a.V + (a.db ? a.V : 0);
    const unsigned grid = (unsigned)std::min<int64_t>(cdiv(n, 256), 8192);
    hipLaunchKernelGGL(round_dw_bf16_kernel, dim3(grid), dim3(256), 0, st, static_cast<const float*>(b.dW), a.d, a.V,
                       static_cast<uint16_t*>(a.dW), a.lddw, a.dW_beta, static_cast<const float*>(b.db),
                       static_cast<uint16_t*>(a.db));
    return hipGetLastError();
}

hipError_t launch_head_vjp_f32(const HeadVjpArgs& a, hipStream_t st) {
    const VjpWs L = vjp_ws(a.N, a.d, a.V, a.dt);
    Plan p = make_plan(a.N, a.d, a.V, a.dt);
    char* base = static_cast<char*>(a.ws);
    float* cq = reinterpret_cast<float*>(base + L.cq_off);
    float* cqp = reinterpret_cast<float*>(base + L.cqp_off);
    float* vmask = reinterpret_cast<float*>(base + L.vmask_off);
    float* scal = reinterpret_cast<float*>(base + L.scal_off);
    float* hpart = reinterpret_cast<float*>(base + L.hpart_off);
    float* hsum = reinterpret_cast<float*>(base + L.hsum_off);
    float* u = reinterpret_cast<float*>(base + L.u_off);
    float* upart = reinterpret_cast<float*>(base + L.upart_off);
    float* part = reinterpret_cast<float*>(base + L.part_off);
    float* zc = reinterpret_cast<float*>(base + L.zc_off);
    const bool zin = !a.is_residual;   // the R argument holds the logits Z

    // MFMA kernels stage 16-byte rows: leading dimensions multiples of 8 and 16-byte bases;
    // otherwise the SIMT kernels (same plan shape, SIMT tiles) run.
    auto al = [](const void* ptr, int64_t ld) { return reinterpret_cast<uintptr_t>(ptr) % 16 == 0 && ld % 8 == 0; };
    if (a.dt == BOM_BF16 && !(al(a.H, a.ldh) && al(a.W, a.ldw) && al(a.R, a.ldr))) {
        // SIMT tiles with their own k splits over every tile (the workspace covers their partials too)
        p = simt_plan(a.N, a.d, a.V);
    }
    if (L.part_off + partial_bytes(p, a.N, a.d, a.V) > L.total) return hipErrorInvalidValue;   // never taken
    if (!a.dH) p.h.kind = kSimt;   // no dH: no rank-1 vector for it

    // small fp32 heads (at most 64 tiles of 64 x 64 in both products, k ranges up to 8192): one launch
    if (a.dt == BOM_F32) {
        const int64_t tw = cdiv(a.d, SB) * cdiv(a.V, SB), th = a.dH ? cdiv(a.N, SB) * cdiv(a.d, SB) : 0;
        if (tw + th <= 64 && a.N <= 8192 && a.V <= 8192) {
            SmallF32Args sa{static_cast<const float*>(a.H), a.ldh, static_cast<const float*>(a.W), a.ldw,
                            static_cast<const float*>(a.R), a.ldr, zin ? a.row_lse : nullptr, a.labels, a.ignore_index,
                            a.q_hat, a.s, a.n_valid, a.lambda, a.N, a.d, a.V, static_cast<float*>(a.dW), a.lddw,
                            a.dW_beta, static_cast<float*>(a.db), a.dH, a.lddh, a.dh_dt == BOM_BF16 ? 1 : 0,
                            (int)cdiv(a.V, SB), (int)tw, (int)cdiv(a.d, SB)};
            hipLaunchKernelGGL(vjp_small_f32_kernel, dim3((unsigned)(tw + th)), dim3(256), 0, st, sa);
            return hipGetLastError();
        }
    }

    // small products (both on the 128-tile kernel): one fused launch, nothing staged beforehand
    const PlanOverride& ov = plan_override();
    const bool fits31 = ((int64_t)(a.N - 1) * a.ldh + a.d) * 2 < (1LL << 31) &&
                        ((int64_t)(a.N - 1) * a.ldr + a.V) * 2 < (1LL << 31) &&
                        ((int64_t)(a.d - 1) * a.ldw + a.V) * 2 < (1LL << 31);
    // (each tile runs over the whole k range, so both k extents stay short)
    if (a.dt == BOM_BF16 && p.w.kind == kMfma128 && (!a.dH || p.h.kind == kMfma128) && fits31 && a.N <= 8192 &&
        a.V <= 8192 && ov.kw != 1 && ov.kh != 1) {
        FusedArgs fa;
        fa.H = static_cast<const uint16_t*>(a.H);
        fa.ldh = a.ldh;
        fa.W = static_cast<const uint16_t*>(a.W);
        fa.ldw = a.ldw;
        fa.R = static_cast<const uint16_t*>(a.R);
        fa.ldr = a.ldr;
        fa.labels = a.labels;
        fa.ig = a.ignore_index;
        fa.q_hat = a.q_hat;
        fa.s = a.s;
        fa.n_valid = a.n_valid;
        fa.lambda = a.lambda;
        fa.N = a.N;
        fa.d = a.d;
        fa.V = a.V;
        fa.dW = static_cast<float*>(a.dW);
        fa.lddw = a.lddw;
        fa.beta = a.dW_beta;
        fa.dH = a.dH;
        fa.lddh = a.lddh;
        fa.dh_bf16 = a.dh_dt == BOM_BF16;
        fa.db = static_cast<float*>(a.db);
        fa.tw_n = (int)cdiv(a.V, FB);
        fa.tw = (int)cdiv(a.d, FB) * fa.tw_n;
        fa.th_n = (int)cdiv(a.d, FB);
        fa.row_lse = zin ? a.row_lse : nullptr;
        const int th = a.dH ? (int)cdiv(a.N, FB) * fa.th_n : 0;
        hipLaunchKernelGGL(vjp_fused_small_kernel, dim3((unsigned)(fa.tw + th)), dim3(256), 0, st, fa);
        return hipGetLastError();
    }

    // rank-1 vectors first: u for dH, row-block partial sums of H over I for dW (lambda = 0: no history
    // term, so neither is needed and the epilogues add nothing)
    hipError_t e;
    const bool hist = a.lambda != 0.f;
    const bool rw = p.w.kind == kRank1 && hist, rh = p.h.kind == kRank1 && hist;
    const int nrb = (int)cdiv(a.N, kHsRows);
    const int uch = u_chunks(a.d, a.V), ucw = u_chunk_cols(a.d, a.V);
    if (rw || rh) {
        const int nu = rh ? (int)cdiv(std::min<int64_t>((int64_t)a.d * uch, kUWaves), 4) : 0;
        const int ns = rw ? (int)cdiv(a.d, 512) * nrb : 0;
        hipLaunchKernelGGL(vjp_rank1_kernel, dim3((unsigned)(nu + ns)), dim3(256), 0, st,
                           static_cast<const uint16_t*>(a.W), a.ldw, a.d, a.V, a.q_hat, nu, uch, ucw,
                           static_cast<const uint16_t*>(a.H), a.ldh, a.N, a.labels, a.ignore_index, upart, hpart);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    int nprep = a.V > a.N ? a.V : a.N;
    if (nprep < a.d) nprep = a.d;
    hipLaunchKernelGGL(vjp_prep_kernel, dim3((nprep + 255) / 256), dim3(256), 0, st, a.q_hat, a.s, a.n_valid, a.lambda,
                       a.V, a.N, a.labels, a.ignore_index, cq, cqp, vmask, scal, static_cast<float*>(a.db),
                       rw ? hpart : nullptr, nrb, a.d, hsum, zin ? a.row_lse : nullptr, zc, rh ? upart : nullptr, uch, u);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const Fold f{cq, vmask, scal, cqp, zin ? zc : nullptr, a.labels};

    if (p.pair && a.dH && p.w.kind == kRank1 && p.h.kind == kRank1) {
        // one grid: dH's units (k split p.h.splits) first, then dW's tiles over the full k range
        const int inner = (int)cdiv(a.d, LB);
        const int oh = (int)cdiv(a.N, LB), ow = (int)cdiv(a.V, LB);
        const int sh = p.h.splits;
        const int kps_h = (int)(cdiv(cdiv(a.V, sh), WKT) * WKT);
        const int kps_w = (int)(cdiv(a.N, WKT) * WKT);
        const uint16_t* H16 = static_cast<const uint16_t*>(a.H);
        const uint16_t* R16 = static_cast<const uint16_t*>(a.R);
        const uint16_t* W16 = static_cast<const uint16_t*>(a.W);
        const TileRange trh{inner, 0, oh, sh, 0, 0, a.d, (int64_t)a.N * a.d};
        const TileRange trw{inner, 0, ow, 1, 0, 0, 0, 0};
        const WideArgs wh{R16, a.ldr, W16, a.ldw, a.N, a.d, a.V, kps_h, trh, f.scal, hist ? vmask : nullptr, u, a.dH, a.lddh, 0.f,
                          sh > 1 ? part : nullptr, nullptr, f.zc, a.labels};
        const WideArgs ww{H16, a.ldh, R16, a.ldr, a.d, a.V, a.N, kps_w, trw, f.scal, hist ? hsum : nullptr, cq, a.dW, a.lddw,
                          a.dW_beta, nullptr, nullptr, f.zc, a.labels};
        const int nh = (int)(cdiv((int64_t)oh * sh, 8) * 8 * inner);
        const int nw = (int)(cdiv(ow, 8) * 8 * inner);
        const dim3 grid((unsigned)(nh + nw));
        const bool w8 = wave_cfg().pair == 8;
        if (zin) {   // logits input: eight waves
            if (a.dh_dt == BOM_BF16)
                hipLaunchKernelGGL((lds256w_pair_kernel<uint16_t, 8, true>), grid, dim3(512), 0, st, wh, ww, nh);
            else
                hipLaunchKernelGGL((lds256w_pair_kernel<float, 8, true>), grid, dim3(512), 0, st, wh, ww, nh);
        } else if (a.dh_dt == BOM_BF16) {
            if (w8)
                hipLaunchKernelGGL((lds256w_pair_kernel<uint16_t, 8>), grid, dim3(512), 0, st, wh, ww, nh);
            else
                hipLaunchKernelGGL((lds256w_pair_kernel<uint16_t, 4>), grid, dim3(256), 0, st, wh, ww, nh);
        } else {
            if (w8)
                hipLaunchKernelGGL((lds256w_pair_kernel<float, 8>), grid, dim3(512), 0, st, wh, ww, nh);
            else
                hipLaunchKernelGGL((lds256w_pair_kernel<float, 4>), grid, dim3(256), 0, st, wh, ww, nh);
        }
        if ((e = hipGetLastError()) != hipSuccess || sh == 1) return e;
        const int64_t MN = (int64_t)a.N * a.d;
        if (a.dh_dt == BOM_BF16)
            hipLaunchKernelGGL(splitk_rank1_kernel<uint16_t>, dim3((unsigned)cdiv(MN, 256)), dim3(256), 0, st, part, sh,
                               a.N, a.d, 0, 0, hist ? vmask : nullptr, u, static_cast<uint16_t*>(a.dH), a.lddh, 0.f);
        else
            hipLaunchKernelGGL(splitk_rank1_kernel<float>, dim3((unsigned)cdiv(MN, 256)), dim3(256), 0, st, part, sh, a.N,
                               a.d, 0, 0, hist ? vmask : nullptr, u, static_cast<float*>(a.dH), a.lddh, 0.f);
        return hipGetLastError();
    }

    // dW = H^T G
    e = run_gemm<float>(true, p.w, a.H, a.ldh, a.R, a.ldr, a.dt, a.d, a.V, a.N, f, static_cast<float*>(a.dW), a.lddw,
                        a.dW_beta, part, hist ? hsum : nullptr, cq,
                        st);
    if (e != hipSuccess) return e;
    // dH = G W^T (shares the split-K buffer: same stream, so it runs after the dW reduction)
    if (a.dH) {
        if (a.dh_dt == BOM_BF16)
            return run_gemm<uint16_t>(false, p.h, a.R, a.ldr, a.W, a.ldw, a.dt, a.N, a.d, a.V, f,
                                      static_cast<uint16_t*>(a.dH), a.lddh, 0.f, part, hist ? vmask : nullptr, u, st);
        return run_gemm<float>(false, p.h, a.R, a.ldr, a.W, a.ldw, a.dt, a.N, a.d, a.V, f, static_cast<float*>(a.dH),
                               a.lddh, 0.f, part, hist ? vmask : nullptr, u, st);
    }
    return hipSuccess;
}

// ---- head forward (support): Z = H W + b, fp32 SIMT ------------------------------------------------
namespace {
// SIMT forward (fp32, and bf16 shapes the MFMA tiles do not take): 64 x 64 tiles, 16-deep k, fp32
// accumulation, Z rounded once to its type.
template <typename T>
__global__ __launch_bounds__(256) void head_forward_simt_kernel(const T* __restrict__ H, int64_t ldh,
                                                                const T* __restrict__ W, int64_t ldw,
                                                                const T* __restrict__ b, int N, int d, int V,
                                                                T* __restrict__ Z, int64_t ldz) {
    __shared__ float As[SK][SB + 4];
    __shared__ float Bs[SK][SB + 4];
    const int t = threadIdx.x, tx = t % 16, ty = t / 16;
    const int m0 = blockIdx.y * SB, n0 = blockIdx.x * SB;
    float acc[4][4] = {};
    for (int k0 = 0; k0 < d; k0 += SK) {
        for (int e = 0; e < 4; ++e) {
            const int idx = e * 256 + t;
            const int rr = idx / SK, kk = idx % SK;
            As[kk][rr] = (k0 + kk < d && m0 + rr < N) ? ldf<T>(H, (int64_t)(m0 + rr) * ldh + k0 + kk) : 0.f;
            const int kk2 = idx / SB, cc = idx % SB;
            Bs[kk2][cc] = (k0 + kk2 < d && n0 + cc < V) ? ldf<T>(W, (int64_t)(k0 + kk2) * ldw + n0 + cc) : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < SK; ++kk) {
            float a4[4], b4[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a4[i] = As[kk][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) b4[j] = Bs[kk][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a4[i], b4[j], acc[i][j]);
        }
        __syncthreads();
    }
    for (int i = 0; i < 4; ++i)
        for (int j = 0; j < 4; ++j) {
            const int m = m0 + ty * 4 + i, n = n0 + tx * 4 + j;
            if (m < N && n < V) stf<T>(Z, (int64_t)m * ldz + n, acc[i][j] + (b ? ldf<T>(b, n) : 0.f));
        }
}
}  // namespace

hipError_t launch_head_forward(const void* H, int64_t ldh, const void* W, int64_t ldw, const void* b, bom_dtype dt,
                               int N, int d, int V, void* Z, int64_t ldz, hipStream_t st) {
    if (dt == BOM_F32) {
        dim3 grid((V + SB - 1) / SB, (N + SB - 1) / SB);
        hipLaunchKernelGGL(head_forward_simt_kernel<float>, grid, dim3(256), 0, st, static_cast<const float*>(H), ldh,
                           static_cast<const float*>(W), ldw, static_cast<const float*>(b), N, d, V,
                           static_cast<float*>(Z), ldz);
        return hipGetLastError();
    }
    const uint16_t* H16 = static_cast<const uint16_t*>(H);
    const uint16_t* W16 = static_cast<const uint16_t*>(W);
    const uint16_t* b16 = static_cast<const uint16_t*>(b);
    auto al = [](const void* ptr, int64_t ld) { return reinterpret_cast<uintptr_t>(ptr) % 16 == 0 && ld % 8 == 0; };
    // 256-tile MFMA kernel: 16-byte chunks along H's rows (k = d) and W's rows (n = V)
    if (d % 8 == 0 && V % 8 == 0 && al(H, ldh) && al(W, ldw) &&
        ((int64_t)(N - 1) * ldh + d) * 2 < (1LL << 31) && ((int64_t)(d - 1) * ldw + V) * 2 < (1LL << 31)) {
        const int MT = (int)cdiv(N, LB), NT = (int)cdiv(V, LB);
        const TileRange tr{MT, 0, NT, 1, 0, 0, 0, 0, xcd_blocked(MT)};
        const WideArgs wa{H16, ldh, W16, ldw, N, V, d, (int)(cdiv(d, WKT) * WKT), tr, nullptr, nullptr, nullptr, Z, ldz,
                          0.f, nullptr, b16};
        const dim3 grid((unsigned)(cdiv(NT, 8) * 8 * MT));
        if (wave_cfg().fwd == 8)
            hipLaunchKernelGGL((lds256w_fwd_kernel<uint16_t, 8>), grid, dim3(512), 0, st, wa);
        else
            hipLaunchKernelGGL((lds256w_fwd_kernel<uint16_t, 4>), grid, dim3(256), 0, st, wa);
        return hipGetLastError();
    }
    dim3 grid((V + SB - 1) / SB, (N + SB - 1) / SB);
    hipLaunchKernelGGL(head_forward_simt_kernel<uint16_t>, grid, dim3(256), 0, st, H16, ldh, W16, ldw, b16, N, d, V,
                       static_cast<uint16_t*>(Z), ldz);
    return hipGetLastError();
}

bool head_forward_stats_supported(const void* H, int64_t ldh, const void* W, int64_t ldw, const void* Z, int64_t ldz,
                                  int N, int d, int V) {
    auto al = [](const void* ptr, int64_t ld) { return reinterpret_cast<uintptr_t>(ptr) % 16 == 0 && ld % 8 == 0; };
    return d % 8 == 0 && V % 8 == 0 && al(H, ldh) && al(W, ldw) && al(Z, ldz) &&
           ((int64_t)(N - 1) * ldh + d) * 2 < (1LL << 31) && ((int64_t)(d - 1) * ldw + V) * 2 < (1LL << 31);
}

hipError_t launch_head_forward_stats(const void* H, int64_t ldh, const void* W, int64_t ldw, const void* b, int N, int d,
                                     int V, void* Z, int64_t ldz, const int32_t* labels, int32_t ignore_index,
                                     float* stats, float* row_target, hipStream_t st) {
    if (!head_forward_stats_supported(H, ldh, W, ldw, Z, ldz, N, d, V)) return hipErrorInvalidValue;
    const int MT = (int)cdiv(N, LB), NT = (int)cdiv(V, LB);
    const TileRange tr{MT, 0, NT, 1, 0, 0, 0, 0, xcd_blocked(MT)};
    WideArgs wa{static_cast<const uint16_t*>(H), ldh, static_cast<const uint16_t*>(W), ldw, N, V, d,
                (int)(cdiv(d, WKT) * WKT), tr, nullptr, nullptr, nullptr, Z, ldz, 0.f, nullptr,
                static_cast<const uint16_t*>(b)};
    wa.stats = stats;
    wa.stats_ld = NT;
    wa.labels = labels;
    wa.ignore_index = ignore_index;
    wa.row_target = row_target;
    hipLaunchKernelGGL((lds256w_fwd_kernel<uint16_t, 8, true>), dim3((unsigned)(cdiv(NT, 8) * 8 * MT)), dim3(512), 0, st, wa);
    return hipGetLastError();
}

}  // namespace bom
