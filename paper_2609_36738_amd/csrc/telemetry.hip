// bom_head_telemetry kernels: historical-projection drift of the linear head (Sec. 3.3, Eq. (8);
// appendix "Measuring historical projection drift"). A diagnostic beside the four steps, for telemetry
// steps only. With hbar = (1/N_t) sum_{i in I} H_i, one call computes
//   M_W = beta1 M_W + (1 - beta1) hbar s^T,  M_b = beta1 M_b + (1 - beta1) s   (own-step projections)
//   Mhat = M / (1 - beta1^t),  h = (hbar q_hat^T, q_hat)                     (BOM's reprojection)
// and reports cos(Mhat, h), ||Mhat - h|| / ||Mhat||, the within-batch cancellation
// ||s|| / ((1/N_t) sum_{i in I} ||r_i||), ||Mhat|| and ||h||.
// Launches: (1) column partial sums of H over valid rows, and residual row norms; (2) hbar; (3) one
// workgroup per row of M_W (and one for M_b): the EMA in place and four fp64 sums; (4) one workgroup
// finishes the statistics. Every sum runs in a fixed order (deterministic).
#include "common.hpp"
#include "kernels.hpp"

namespace bom {
namespace {

constexpr int kTeleRows = 128;   // rows of H per column-sum block
constexpr int kNormBlocks = 2048; // blocks of the residual row-norm pass (four waves, one row each at a time)

template <typename T>
__device__ __forceinline__ float ldv(const T* p, int64_t i);
template <>
__device__ __forceinline__ float ldv<float>(const float* p, int64_t i) { return p[i]; }
template <>
__device__ __forceinline__ float ldv<uint16_t>(const uint16_t* p, int64_t i) { return bf16_to_f32(p[i]); }

// Blocks [0, nhb): block (cb, rb) adds rows [rb * kTeleRows, +kTeleRows) of H over I for the 256 columns
// of cb (thread t: column cb * 256 + t), in row order. Blocks [nhb, nhb + kNormBlocks): each wave takes
// rows w, w + W, ... of R and adds ||r_i|| over valid rows; the block sum goes to rpart (fp64).
template <typename TH, typename TR>
__global__ __launch_bounds__(256) void tele_stats_kernel(const TH* __restrict__ H, int64_t ldh, const TR* __restrict__ R,
                                                         int64_t ldr, int N, int d, int V,
                                                         const int32_t* __restrict__ labels, int32_t ignore_index,
                                                         int ncb, int nhb, float* __restrict__ hpart,
                                                         double* __restrict__ rpart) {
    __shared__ double sh[4];
    const int t = threadIdx.x;
    if ((int)blockIdx.x < nhb) {
        const int cb = blockIdx.x % ncb, rb = blockIdx.x / ncb;
        const int k = cb * 256 + t;
        if (k >= d) return;
        float acc = 0.f;
        const int r1 = min(N, (rb + 1) * kTeleRows);
        for (int i = rb * kTeleRows; i < r1; ++i) {
            bool bad = false;
            if (label_valid(labels[i], V, ignore_index, &bad)) acc += ldv<TH>(H, (int64_t)i * ldh + k);
        }
        hpart[(int64_t)rb * d + k] = acc;
        return;
    }
    const int b = blockIdx.x - nhb;
    const int lane = t % kWave, w = t / kWave;
    // 16-byte groups (8 bf16 or 4 fp32) when every row starts 16-byte aligned, the rest element-wise
    constexpr int G = 16 / sizeof(TR);
    const bool vec = reinterpret_cast<uintptr_t>(R) % 16 == 0 && (ldr * sizeof(TR)) % 16 == 0;
    const int nvec = vec ? V / G : 0;
    double sum = 0.0;
    for (int i = b * 4 + w; i < N; i += kNormBlocks * 4) {
        bool bad = false;
        if (!label_valid(labels[i], V, ignore_index, &bad)) continue;   // wave-uniform
        const TR* row = R + (int64_t)i * ldr;
        float rr = 0.f;
        auto add = [&](const u32x4_t& x) {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                if constexpr (sizeof(TR) == 2) {
                    const float lo = bf16_lo(x[c]), hi = bf16_hi(x[c]);
                    rr = fmaf(lo, lo, fmaf(hi, hi, rr));
                } else {
                    const float f = __uint_as_float(x[c]);
                    rr = fmaf(f, f, rr);
                }
            }
        };
        const u32x4_t* rv = reinterpret_cast<const u32x4_t*>(row);
        int q = lane;
        for (; q + 3 * kWave < nvec; q += 4 * kWave) {   // four 16-byte loads in flight per lane
            u32x4_t x[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) x[k] = __builtin_nontemporal_load(rv + q + k * kWave);
#pragma unroll
            for (int k = 0; k < 4; ++k) add(x[k]);
        }
        for (; q < nvec; q += kWave) add(__builtin_nontemporal_load(rv + q));
        for (int j = nvec * G + lane; j < V; j += kWave) {
            const float x = ldv<TR>(row, j);
            rr = fmaf(x, x, rr);
        }
        rr = wave_sum(rr);
        sum += sqrt((double)rr);
    }
    if (lane == 0) sh[w] = sum;
    __syncthreads();
    if (t == 0) rpart[b] = ((sh[0] + sh[1]) + sh[2]) + sh[3];
}

// hbar_k = (sum over row blocks of hpart[rb][k]) / N_t, in row-block order (0 when N_t = 0).
__global__ __launch_bounds__(256) void tele_hbar_kernel(const float* __restrict__ hpart, int nrb, int d,
                                                        const int32_t* __restrict__ n_valid, float* __restrict__ hbar) {
    const int k = blockIdx.x * 256 + threadIdx.x;
    if (k >= d) return;
    float a = 0.f;
    for (int rb = 0; rb < nrb; ++rb) a += hpart[(int64_t)rb * d + k];
    const int nt = *n_valid;
    hbar[k] = nt > 0 ? a / (float)nt : 0.f;
}

// Block k < d: row k of M_W; block d: M_b (when present). The EMA in place, then the sums
// (||Mhat||^2, <Mhat, h>, ||h||^2, ||Mhat - h||^2) of the row in fp64, written to mpart[block][4].
__global__ __launch_bounds__(256) void tele_m_kernel(float* __restrict__ MW, int64_t ldm, float* __restrict__ Mb,
                                                     int d, int V, const float* __restrict__ hbar,
                                                     const float* __restrict__ s, const float* __restrict__ q_hat,
                                                     float beta1, float one_minus_beta1, float inv_bc,
                                                     double* __restrict__ mpart) {
    __shared__ double sh[4][4];
    const int t = threadIdx.x;
    const int k = blockIdx.x;
    float* row = k < d ? MW + (int64_t)k * ldm : Mb;
    const float hk = k < d ? hbar[k] : 1.f;   // the bias block projects through the identity
    double mm = 0.0, mh = 0.0, hh = 0.0, dd = 0.0;
    auto one = [&](float mold, float sj, float qj) {
        const float m = fmaf(beta1, mold, one_minus_beta1 * (hk * sj));
        const double mhat = (double)m * inv_bc, hv = (double)hk * qj;
        mm += mhat * mhat;
        mh += mhat * hv;
        hh += hv * hv;
        dd += (mhat - hv) * (mhat - hv);
        return m;
    };
    // 16-byte groups where row, s and q_hat allow it, the rest element-wise
    const bool vec = reinterpret_cast<uintptr_t>(row) % 16 == 0 && reinterpret_cast<uintptr_t>(s) % 16 == 0 &&
                     reinterpret_cast<uintptr_t>(q_hat) % 16 == 0;
    const int nvec = vec ? V / 4 : 0;
    for (int q = t; q < nvec; q += 256) {
        f32x4 m4 = ld_stream(row + q * 4);
        const f32x4 s4 = *reinterpret_cast<const f32x4*>(s + q * 4);
        const f32x4 q4 = *reinterpret_cast<const f32x4*>(q_hat + q * 4);
#pragma unroll
        for (int c = 0; c < 4; ++c) m4[c] = one(m4[c], s4[c], q4[c]);
        st_stream(row + q * 4, m4);
    }
    for (int j = nvec * 4 + t; j < V; j += 256) row[j] = one(row[j], s[j], q_hat[j]);
    mm = wave_sum(mm);
    mh = wave_sum(mh);
    hh = wave_sum(hh);
    dd = wave_sum(dd);
    const int lane = t % kWave, w = t / kWave;
    if (lane == 0) {
        sh[w][0] = mm;
        sh[w][1] = mh;
        sh[w][2] = hh;
        sh[w][3] = dd;
    }
    __syncthreads();
    if (t < 4) mpart[(int64_t)k * 4 + t] = ((sh[0][t] + sh[1][t]) + sh[2][t]) + sh[3][t];
}

// One block: the sums over rows (block order), ||s||, the mean residual row norm, and the outputs.
__global__ __launch_bounds__(256) void tele_finish_kernel(const double* __restrict__ mpart, int nm,
                                                          const double* __restrict__ rpart, const float* __restrict__ s,
                                                          int V, const int32_t* __restrict__ n_valid,
                                                          float* __restrict__ out) {
    __shared__ double sh[6][256];
    const int t = threadIdx.x;
    double a[6] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
    for (int k = t; k < nm; k += 256)
        for (int c = 0; c < 4; ++c) a[c] += mpart[(int64_t)k * 4 + c];
    for (int b = t; b < kNormBlocks; b += 256) a[4] += rpart[b];
    for (int j = t; j < V; j += 256) a[5] += (double)s[j] * s[j];
    for (int c = 0; c < 6; ++c) sh[c][t] = a[c];
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if (t < o)
            for (int c = 0; c < 6; ++c) sh[c][t] += sh[c][t + o];
        __syncthreads();
    }
    if (t == 0) {
        const double mm = sh[0][0], mh = sh[1][0], hh = sh[2][0], dd = sh[3][0];
        const int nt = *n_valid;
        const double rmean = nt > 0 ? sh[4][0] / nt : 0.0;
        out[0] = (float)(mm > 0.0 && hh > 0.0 ? mh / (sqrt(mm) * sqrt(hh)) : 0.0);
        out[1] = (float)(mm > 0.0 ? sqrt(dd) / sqrt(mm) : 0.0);
        out[2] = (float)(rmean > 0.0 ? sqrt(sh[5][0]) / rmean : 0.0);
        out[3] = (float)sqrt(mm);
        out[4] = (float)sqrt(hh);
    }
}

struct TeleLayout {
    int ncb, nrb;
    size_t hpart_off, hbar_off, rpart_off, mpart_off, total;
};

TeleLayout tele_layout(int64_t N, int64_t d) {
    TeleLayout L;
    L.ncb = (int)((d + 255) / 256);
    L.nrb = (int)((N + kTeleRows - 1) / kTeleRows);
    L.hpart_off = 0;
    L.hbar_off = align256((size_t)L.nrb * d * 4);
    L.rpart_off = align256(L.hbar_off + (size_t)d * 4);
    L.mpart_off = align256(L.rpart_off + (size_t)kNormBlocks * 8);
    L.total = align256(L.mpart_off + (size_t)(d + 1) * 4 * 8);
    return L;
}

template <typename TH, typename TR>
hipError_t launch_stats(const TeleArgs& a, const TeleLayout& L, char* ws, hipStream_t st) {
    const int nhb = L.ncb * L.nrb;
    hipLaunchKernelGGL((tele_stats_kernel<TH, TR>), dim3((unsigned)(nhb + kNormBlocks)), dim3(256), 0, st,
                       static_cast<const TH*>(a.H), a.ldh, static_cast<const TR*>(a.R), a.ldr, a.N, a.d, a.V, a.labels,
                       a.ignore_index, L.ncb, nhb, reinterpret_cast<float*>(ws + L.hpart_off),
                       reinterpret_cast<double*>(ws + L.rpart_off));
    return hipGetLastError();
}

}  // namespace

size_t head_telemetry_workspace_bytes(int64_t N, int64_t d) { return tele_layout(N, d).total; }

hipError_t launch_head_telemetry(const TeleArgs& a, hipStream_t st) {
    const TeleLayout L = tele_layout(a.N, a.d);
    char* ws = static_cast<char*>(a.ws);
    hipError_t e;
    if (a.h_dt == BOM_BF16)
        e = a.r_dt == BOM_BF16 ? launch_stats<uint16_t, uint16_t>(a, L, ws, st) : launch_stats<uint16_t, float>(a, L, ws, st);
    else
        e = a.r_dt == BOM_BF16 ? launch_stats<float, uint16_t>(a, L, ws, st) : launch_stats<float, float>(a, L, ws, st);
    if (e != hipSuccess) return e;
    float* hbar = reinterpret_cast<float*>(ws + L.hbar_off);
    hipLaunchKernelGGL(tele_hbar_kernel, dim3((unsigned)L.ncb), dim3(256), 0, st,
                       reinterpret_cast<const float*>(ws + L.hpart_off), L.nrb, a.d, a.n_valid, hbar);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int nm = a.d + (a.Mb ? 1 : 0);
    double* mpart = reinterpret_cast<double*>(ws + L.mpart_off);
    hipLaunchKernelGGL(tele_m_kernel, dim3((unsigned)nm), dim3(256), 0, st, a.MW, a.ldm, a.Mb, a.d, a.V, hbar, a.s,
                       a.q_hat, a.beta1, a.one_minus_beta1, a.inv_bc, mpart);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(tele_finish_kernel, dim3(1), dim3(256), 0, st, mpart, nm,
                       reinterpret_cast<const double*>(ws + L.rpart_off), a.s, a.V, a.n_valid, a.out);
    return hipGetLastError();
}

}  // namespace bom
