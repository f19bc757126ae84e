// bom_residual kernels: per-row softmax statistics, the residual rows R = softmax(Z) - onehot(y)
// and the batch-mean residual s over the valid rows (Algorithm 1, s_t; Sec. 3.2; the
// token-level appendix for ignored targets).
//
// Three paths, all deterministic (fixed reduction orders, no floating-point atomics):
//  * single pass (V up to ~53k bf16 / ~26k fp32): one persistent workgroup per CU keeps a whole
//    row in registers or LDS, reduces max / argmax / sum across the workgroup, writes R, and
//    accumulates its rows' residuals per column in registers; Z is read from HBM exactly once.
//  * split rows (bf16 up to 524,288 columns): several workgroups share each row and exchange their
//    per-part statistics; Z is still read once.
//  * two pass (other shapes): a stats kernel (one wave per row, online max / sum / argmax) writes the
//    row statistics, then a column-slab kernel re-reads Z, writes R and accumulates per-column
//    partials for blocks of rows.
// A finish step sums the per-workgroup partials in a fixed order into s, loss, N_t and flags.
#include <climits>
#include <cmath>
#include <cstdlib>
#include <mutex>
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "vec_io.hpp"

namespace bom {
namespace {

constexpr int kSingleMaxWG = 256;     // persistent workgroups of the single pass (one per CU)
constexpr int kStatsRowsPerWG = 4;    // two pass, stats: one wave per row, 4 waves per workgroup
constexpr int kColsThreads = 256;     // two pass, columns: threads per workgroup
constexpr int kColsCPT = 8;           // two pass, columns: chunks per thread
constexpr int kColsMaxRowBlock = 256; // two pass, columns: at most this many rows per partial-sum block
constexpr int kSplitMaxParts = 16;    // split rows: at most this many workgroups share a row
constexpr int kSplitMaxNch = 4;       // split rows: 1024 threads x 4 chunks x 8 = 32768 columns per part

// Rows per column-kernel workgroup: enough workgroups (about 1024) to fill the chip.
int cols_row_block(int64_t N, int64_t V, int vec) {
    const int64_t slab = (int64_t)kColsThreads * kColsCPT * vec;
    const int64_t nslab = (V + slab - 1) / slab;
    int64_t rb = (N * nslab + 1023) / 1024;
    if (rb < 8) rb = 8;
    if (rb > kColsMaxRowBlock) rb = kColsMaxRowBlock;
    return (int)rb;
}

struct Partials {
    float* part;      // [nparts][V] per-workgroup column sums of residual rows
    int* wg_count;    // [nwg] valid rows
    int* wg_flags;    // [nwg] BOM_FLAG_LABEL_RANGE bits
    double* wg_loss;  // [nwg] sum of per-row cross-entropy
    unsigned long long* xch;  // [N][S][3] split rows: per-part (max, sum, argmax) records
};

struct WsLayout {
    size_t part_off, count_off, flags_off, loss_off, xch_off, total;
};

bool plan_split(int V, int* S, int* W, int* nch);

WsLayout ws_layout(int64_t N, int64_t V) {
    int64_t nwg1 = N < kSingleMaxWG ? N : kSingleMaxWG;
    int64_t nstats = (N + kStatsRowsPerWG - 1) / kStatsRowsPerWG;
    // the vector width is not known here; a width of 1 gives the most partial-sum blocks
    const int64_t rb = cols_row_block(N, V, 1) < cols_row_block(N, V, 8) ? cols_row_block(N, V, 1)
                                                                         : cols_row_block(N, V, 8);
    int64_t nrb = (N + rb - 1) / rb;
    int64_t nparts = nwg1 > nrb ? nwg1 : nrb;
    int64_t nwg = nwg1 > nstats ? nwg1 : nstats;
    if (nwg < kSingleMaxWG) nwg = kSingleMaxWG;   // split rows: up to kSingleMaxWG workgroups at any N
    WsLayout L;
    L.part_off = 0;
    L.count_off = align256(L.part_off + (size_t)nparts * (size_t)V * sizeof(float));
    L.flags_off = align256(L.count_off + (size_t)nwg * sizeof(int));
    L.loss_off = align256(L.flags_off + (size_t)nwg * sizeof(int));
    L.xch_off = align256(L.loss_off + (size_t)nwg * sizeof(double));
    int S = 0, W = 0, nch = 0;
    const int64_t xparts = plan_split((int)V, &S, &W, &nch) ? S : 0;
    L.total = align256(L.xch_off + (size_t)N * (size_t)xparts * 3 * sizeof(unsigned long long));
    return L;
}

template <int NW>
__device__ __forceinline__ float block_max(float v, float* sh) {
    v = wave_max_dpp(v);
    if ((threadIdx.x & (kWave - 1)) == 0) sh[threadIdx.x / kWave] = v;
    __syncthreads();
    float r = sh[0];
#pragma unroll
    for (int w = 1; w < NW; ++w) r = fmaxf(r, sh[w]);
    return r;
}
template <int NW>
__device__ __forceinline__ float block_sum(float v, float* sh) {
    v = wave_sum_dpp(v);
    if ((threadIdx.x & (kWave - 1)) == 0) sh[threadIdx.x / kWave] = v;
    __syncthreads();
    float r = sh[0];
#pragma unroll
    for (int w = 1; w < NW; ++w) r += sh[w];
    return r;
}
template <int NW>
__device__ __forceinline__ int block_min(int v, int* sh) {
    v = wave_min_dpp(v);
    if ((threadIdx.x & (kWave - 1)) == 0) sh[threadIdx.x / kWave] = v;
    __syncthreads();
    int r = sh[0];
#pragma unroll
    for (int w = 1; w < NW; ++w) r = min(r, sh[w]);
    return r;
}

template <int VEC>
__device__ __forceinline__ void store_f32_chunk(float* row, int col, int V, const float* x) {
    if (col < V) {
        if (VEC % 4 == 0) {
#pragma unroll
            for (int k = 0; k < VEC; k += 4) VecIO<float, 4>::store(row + col + k, x + k);
        } else {
#pragma unroll
            for (int k = 0; k < VEC; ++k) row[col + k] = x[k];
        }
    }
}

// ---------------------------------------------------------------------------------------------
// Single pass. Thread `tid` owns columns (c * THREADS + tid) * VEC + k, c < NCH, k < VEC.
// PACKED (bf16 only, for wide rows): the row stays as raw bf16 pairs and exp is evaluated twice
// (once for the sum, once for p); otherwise e = exp(z - m) is kept in fp32 registers.
template <typename T, int THREADS, int VEC, int NCH, bool PACKED>
__global__ __launch_bounds__(THREADS) void residual_rows_kernel(
    const T* __restrict__ Z, int64_t ldz, int N, int V, const int32_t* __restrict__ labels, int32_t ignore_index,
    float* __restrict__ row_lse, int32_t* __restrict__ row_argmax, float* __restrict__ row_target,
    T* __restrict__ R, int64_t ldr, int rows_per_wg, Partials ws) {
    constexpr int NW = THREADS / kWave;
    constexpr int VPT = NCH * VEC;
    constexpr int NXW = PACKED ? VPT / 2 : 1;  // raw bf16 pairs (PACKED)
    constexpr int NXF = PACKED ? 1 : VPT;      // fp32 values (otherwise)
    static_assert(!PACKED || (VEC == 8), "packed rows need 16-byte bf16 chunks");
    __shared__ float sh_max[NW];
    __shared__ int sh_idx[NW];
    __shared__ float sh_sum[NW];
    const int tid = threadIdx.x;

    float acc[VPT];
#pragma unroll
    for (int k = 0; k < VPT; ++k) acc[k] = 0.f;

    const int row0 = blockIdx.x * rows_per_wg;
    const int row1 = min(row0 + rows_per_wg, N);
    int cnt = 0;
    double ce = 0.0;
    bool bad = false;

    for (int i = row0; i < row1; ++i) {
        const T* zr = Z + (int64_t)i * ldz;
        float x[NXF];
        uint32_t xw[NXW];
        // A chunk whose columns can reach past the row's end is loaded with a bounds check (padding -inf):
        // the last one, and the ones before it when NCH exceeds the row's chunk count (NCH comes from a
        // fixed set of sizes). Uniform across the workgroup.
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int col = (c * THREADS + tid) * VEC;
            const bool last = (c + 1) * THREADS * VEC > V;
            if constexpr (PACKED) {
                const bool ok = !last || col < V;
                const uint4 u = *reinterpret_cast<const uint4*>(zr + (ok ? col : V - VEC));
                if (last) {
                    const uint32_t m = lane_mask(ok), fb = 0xFF80FF80u & ~m;  // padding: a pair of bf16 -inf
                    xw[c * 4 + 0] = (u.x & m) | fb; xw[c * 4 + 1] = (u.y & m) | fb;
                    xw[c * 4 + 2] = (u.z & m) | fb; xw[c * 4 + 3] = (u.w & m) | fb;
                } else {
                    xw[c * 4 + 0] = u.x; xw[c * 4 + 1] = u.y; xw[c * 4 + 2] = u.z; xw[c * 4 + 3] = u.w;
                }
            } else if (last) {
                load_chunk<T, VEC>(zr, col, V, -INFINITY, &x[c * VEC]);
            } else {
                VecIO<T, VEC>::load(zr + col, &x[c * VEC]);
            }
        }
        auto val = [&](int k) -> float {
            if constexpr (PACKED) return (k & 1) ? bf16_hi(xw[k >> 1]) : bf16_lo(xw[k >> 1]);
            else return x[k];
        };

        // max, then the lowest column attaining it
        float tm = -INFINITY;
#pragma unroll
        for (int k = 0; k < VPT; ++k) tm = fmaxf(tm, val(k));
        const float m = block_max<NW>(tm, sh_max);
        int ti = INT_MAX;
        if (tm == m) {
#pragma unroll
            for (int c = NCH - 1; c >= 0; --c)
#pragma unroll
                for (int k = VEC - 1; k >= 0; --k)
                    if (val(c * VEC + k) == m) ti = (c * THREADS + tid) * VEC + k;
        }
        const int am = block_min<NW>(ti, sh_idx);
        if constexpr (PACKED) {
            // keep the row packed: stop the compiler from caching unpacked values across passes
#pragma unroll
            for (int k = 0; k < NXW; ++k) asm volatile("" : "+v"(xw[k]));
        }

        // l = sum exp(z - m)
        const float m2 = m * kLog2e;
        float l = 0.f;
        if constexpr (PACKED) {
#pragma unroll
            for (int k = 0; k < VPT; ++k) l += exp2_fast(fmaf(val(k), kLog2e, -m2));
        } else {
#pragma unroll
            for (int k = 0; k < VPT; ++k) {
                x[k] = exp2_fast(fmaf(x[k], kLog2e, -m2));
                l += x[k];
            }
        }
        l = block_sum<NW>(l, sh_sum);
        const float lse = m + logf(l);
        if constexpr (PACKED) {
#pragma unroll
            for (int k = 0; k < NXW; ++k) asm volatile("" : "+v"(xw[k]));
        }

        const int y = labels[i];
        bool rbad = false;
        const bool valid = label_valid(y, V, ignore_index, &rbad);
        bad |= rbad;
        T* rr = R ? R + (int64_t)i * ldr : nullptr;
        if (valid) {
            // the label column is owned by exactly one thread: subtract the one-hot there
            const int yv = y / VEC;
            const int slot = (yv % THREADS == tid) ? (yv / THREADS) * VEC + (y % VEC) : -1;
            const float inv_l = 1.0f / l;
            const float lse2 = lse * kLog2e;
#pragma unroll
            for (int c = 0; c < NCH; ++c) {
                float p[VEC];
#pragma unroll
                for (int k = 0; k < VEC; ++k) {
                    if constexpr (PACKED) p[k] = exp2_fast(fmaf(val(c * VEC + k), kLog2e, -lse2));
                    else p[k] = x[c * VEC + k] * inv_l;
                }
                if (slot >= 0) {
#pragma unroll
                    for (int k = 0; k < VEC; ++k)
                        if (c * VEC + k == slot) p[k] -= 1.0f;
                }
#pragma unroll
                for (int k = 0; k < VEC; ++k) acc[c * VEC + k] += p[k];
                if (rr) store_chunk<T, VEC>(rr, (c * THREADS + tid) * VEC, V, p);
            }
        } else if (rr) {
            float zero[VEC];
#pragma unroll
            for (int k = 0; k < VEC; ++k) zero[k] = 0.f;
#pragma unroll
            for (int c = 0; c < NCH; ++c) store_chunk<T, VEC>(rr, (c * THREADS + tid) * VEC, V, zero);
        }
        if (tid == 0) {
            row_lse[i] = lse;
            if (row_argmax) row_argmax[i] = am;
            const float zt = valid ? load_scalar<T>(zr + y) : 0.f;
            if (row_target) row_target[i] = zt;
            if (valid) {
                ++cnt;
                ce += (double)lse - (double)zt;
            }
        }
    }

    float* prow = ws.part + (int64_t)blockIdx.x * V;
#pragma unroll
    for (int c = 0; c < NCH; ++c) store_f32_chunk<VEC>(prow, (c * THREADS + tid) * VEC, V, &acc[c * VEC]);
    if (tid == 0) {
        ws.wg_count[blockIdx.x] = cnt;
        ws.wg_loss[blockIdx.x] = ce;
        ws.wg_flags[blockIdx.x] = bad ? BOM_FLAG_LABEL_RANGE : 0;
    }
}

// ---------------------------------------------------------------------------------------------
// Single pass, wide bf16 rows: each thread parks its raw 16-byte chunks in its own LDS slots
// (thread-private) and keeps only its column accumulators in registers. Rows are software-
// pipelined through registers: after the second pass of row i the thread parks row i+1 and loads
// row i+2 into the freed registers, so each row's loads are in flight for a whole row's work.
// Workgroup g takes rows g, g + G, g + 2G, ... so the workgroups sweep the matrix together. The
// row maximum and sum of exp(z - max) come from one online pass over the
// slots (running max with the sum rescaled when it grows), a wave reduction (maximum, then the
// rescaled sums) and one workgroup barrier per row; the argmax comes from the one chunk per thread
// where the thread's maximum first appeared. The second pass forms p = exp(z - lse), the
// residual, the column sums and R. Per-row words shared across the workgroup are double buffered,
// and the previous row's argmax and target logit are written after the next barrier.
template <int THREADS, int NCH>
__global__ __launch_bounds__(THREADS) void residual_rows_lds_kernel(
    const uint16_t* __restrict__ Z, int64_t ldz, int N, int V, const int32_t* __restrict__ labels, int32_t ignore_index,
    float* __restrict__ row_lse, int32_t* __restrict__ row_argmax, float* __restrict__ row_target,
    uint16_t* __restrict__ R, int64_t ldr, int rows_per_wg, Partials ws) {
    constexpr int VEC = 8;
    constexpr int NW = THREADS / kWave;
    constexpr int VPT = NCH * VEC;
    __shared__ uint4 slots[NCH * THREADS];
    __shared__ float sh_m[2][NW];
    __shared__ float sh_l[2][NW];
    __shared__ int sh_am[2];
    __shared__ float sh_zt[2];
    const int tid = threadIdx.x;
    float acc[VPT];
#pragma unroll
    for (int k = 0; k < VPT; ++k) acc[k] = 0.f;
    // rows blockIdx.x + j * gridDim.x (j < nr): the workgroups sweep the matrix together
    const int G = gridDim.x;
    const int nr = blockIdx.x < N ? (N - 1 - (int)blockIdx.x) / G + 1 : 0;
    auto row_of = [&](int j) { return (int)blockIdx.x + j * G; };
    (void)rows_per_wg;
    int cnt = 0;
    double ce = 0.0;
    bool bad = false;
    auto unpack = [](const uint4& u, float* x) {
        x[0] = bf16_lo(u.x); x[1] = bf16_hi(u.x); x[2] = bf16_lo(u.y); x[3] = bf16_hi(u.y);
        x[4] = bf16_lo(u.z); x[5] = bf16_hi(u.z); x[6] = bf16_lo(u.w); x[7] = bf16_hi(u.w);
    };
    // Row loads and R stores go through per-row buffer descriptors: chunk c of this thread sits at
    // byte tid*16 + c*THREADS*16, all of it in the range-checked vector offset, so chunks past the
    // row's end load zeros (replaced by -inf when parked) and their stores are dropped.
    const int voff = tid * 16;
    // the first chunk index of this wave's lanes whose chunks may lie past the row's end
    const int wave_last = (tid | (kWave - 1));
    auto row_desc = [&](int i) { return make_desc(Z + (int64_t)i * ldz, V * 2); };
    auto load_chunk = [&](const __amdgpu_buffer_rsrc_t& d, int c) {
        const u32x4_t w = __builtin_amdgcn_raw_buffer_load_b128(d, voff + c * THREADS * 16, 0, 0);
        return make_uint4(w[0], w[1], w[2], w[3]);
    };
    // park chunk c of a row (chunks past the row's end: bf16 -inf)
    auto park = [&](int c, uint4 w) {
        if ((c * THREADS + wave_last) * VEC >= V) {   // uniform per wave
            const bool ok = ((c * THREADS + tid) * VEC) < V;
            const uint32_t mk = lane_mask(ok), fb = 0xFF80FF80u & ~mk;
            w = make_uint4((w.x & mk) | fb, (w.y & mk) | fb, (w.z & mk) | fb, (w.w & mk) | fb);
        }
        slots[c * THREADS + tid] = w;
    };
    uint4 nxt[NCH];
    if (nr > 0) {
        const auto d0 = row_desc(row_of(0));
#pragma unroll
        for (int c = 0; c < NCH; ++c) nxt[c] = load_chunk(d0, c);
#pragma unroll
        for (int c = 0; c < NCH; ++c) park(c, nxt[c]);
        if (nr > 1) {
            const auto d1 = row_desc(row_of(1));
#pragma unroll
            for (int c = 0; c < NCH; ++c) nxt[c] = load_chunk(d1, c);
        }
    }
    if (tid < 2) sh_am[tid] = INT_MAX;   // first used after the first barrier
    // tid 0 finishes a row's argmax, target logit and loss term after the next row's barrier
    auto finish_row = [&](int i, int b, float lse, bool valid) {
        if (row_argmax) row_argmax[i] = sh_am[b];
        sh_am[b] = INT_MAX;   // reused two rows later, after a barrier this thread has yet to reach
        const float zt = valid ? sh_zt[b] : 0.f;
        if (row_target) row_target[i] = zt;
        if (valid) {
            ++cnt;
            ce += (double)lse - (double)zt;
        }
    };
    float prev_lse = 0.f;
    bool prev_valid = false;
    for (int j = 0; j < nr; ++j) {
        const int i = row_of(j);
        const int b = j & 1;
        // pass 1 (LDS): online (max, sum) over this thread's chunks, in column order, with the
        // first chunk that reached the thread's maximum; the next chunk is read ahead
        float m = -INFINITY, l = 0.f;
        int cmax = 0;
        uint4 u_next = slots[tid];
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const uint4 u = u_next;
            if (c + 1 < NCH) u_next = slots[(c + 1) * THREADS + tid];
            float x[VEC];
            unpack(u, x);
            // IEEE maximum (no canonicalising moves of the unpacked bit patterns)
            auto mx = [](float a, float b2) { return __builtin_elementwise_maximum(a, b2); };
            const float cm = mx(mx(mx(x[0], x[1]), mx(x[2], x[3])), mx(mx(x[4], x[5]), mx(x[6], x[7])));
            const float mn = mx(m, cm);
            // a padding-only chunk after real ones leaves (m, l) unchanged (mn == m, terms zero);
            // chunk 0 of every thread lies inside the row, so mn is finite
            const float mn2 = mn * kLog2e;
            float e[VEC];
#pragma unroll
            for (int k = 0; k < VEC; ++k) e[k] = exp2_fast(fmaf(x[k], kLog2e, -mn2));
            const float cl = ((e[0] + e[1]) + (e[2] + e[3])) + ((e[4] + e[5]) + (e[6] + e[7]));
            l = (c == 0 ? cl : fmaf(l, exp2_fast((m - mn) * kLog2e), cl));
            if (c > 0 && cm > m) cmax = c;
            m = mn;
        }
        const float m_thread = m;
        // wave: the maximum, then the lanes' sums rescaled to it (DPP lane permutes)
        const float mw = wave_max_dpp(m);
        const float lw = wave_sum_dpp(l * exp2_fast((m - mw) * kLog2e));
        if ((tid & (kWave - 1)) == 0) {
            sh_m[b][tid / kWave] = mw;
            sh_l[b][tid / kWave] = lw;
        }
        __syncthreads();
        if (tid == 0 && j > 0) finish_row(row_of(j - 1), b ^ 1, prev_lse, prev_valid);
        // workgroup: the same over the NW wave pairs, lane w of every wave holding pair w (one 16-lane
        // row reduces them); lane 0's result is broadcast
        static_assert(NW <= 16, "the per-wave values fit one 16-lane row");
        {
            const int lane = tid & (kWave - 1);
            const float mg = lane < NW ? sh_m[b][lane] : -INFINITY;
            const float mm = lane_f32(row16_max(mg), 0);
            const float lg = lane < NW ? sh_l[b][lane] * exp2_fast((mg - mm) * kLog2e) : 0.f;
            m = mm;
            l = lane_f32(row16_sum(lg), 0);
        }
        // argmax: the first column holding the row maximum lies in the first chunk where some
        // thread holding that maximum reached it; those threads search that chunk
        if (m_thread == m) {
            float x[VEC];
            unpack(slots[cmax * THREADS + tid], x);
            int k0 = VEC - 1;
#pragma unroll
            for (int k = VEC - 2; k >= 0; --k) k0 = (x[k] == m) ? k : k0;
            atomicMin(&sh_am[b], (cmax * THREADS + tid) * VEC + k0);
        }
        const float lse = m + logf(l);
        const int y = labels[i];
        bool rbad = false;
        const bool valid = label_valid(y, V, ignore_index, &rbad);
        bad |= rbad;
        // R row stores go through a buffer descriptor (no R: an empty range, every store dropped)
        const auto rdesc = make_desc(R ? R + (int64_t)i * ldr : nullptr, R ? V * 2 : 0);
        const bool has_next = j + 1 < nr, has_next2 = j + 2 < nr;
        const auto dn = row_desc(has_next2 ? row_of(j + 2) : i);
        // pass 2 (LDS): p = exp(z - lse), residual, column accumulation, R; the label's owner
        // also publishes the target logit
        const int yv = y / VEC;
        const int slot = (valid && yv % THREADS == tid) ? (yv / THREADS) * VEC + (y % VEC) : -1;
        const float lse2 = lse * kLog2e;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            float p[VEC];
            if (valid) {
                float x[VEC];
                unpack(slots[c * THREADS + tid], x);
#pragma unroll
                for (int k = 0; k < VEC; ++k) p[k] = exp2_fast(fmaf(x[k], kLog2e, -lse2));
                if (slot >= 0) {
#pragma unroll
                    for (int k = 0; k < VEC; ++k)
                        if (c * VEC + k == slot) {
                            p[k] -= 1.0f;
                            sh_zt[b] = x[k];
                        }
                }
#pragma unroll
                for (int k = 0; k < VEC; ++k) acc[c * VEC + k] += p[k];
            } else {
#pragma unroll
                for (int k = 0; k < VEC; ++k) p[k] = 0.f;
            }
            u32x4_t w;
            w[0] = pack_bf16x2(p[0], p[1]);
            w[1] = pack_bf16x2(p[2], p[3]);
            w[2] = pack_bf16x2(p[4], p[5]);
            w[3] = pack_bf16x2(p[6], p[7]);
            __builtin_amdgcn_raw_buffer_store_b128(w, rdesc, voff + c * THREADS * 16, 0, 0);
        }
        if (tid == 0) row_lse[i] = lse;
        // park the next row (its loads were issued before this row's stores, so waiting for them
        // does not wait for the stores) and load the one after into the freed registers
        if (has_next) {
#pragma unroll
            for (int c = 0; c < NCH; ++c) park(c, nxt[c]);
            if (has_next2) {
#pragma unroll
                for (int c = 0; c < NCH; ++c) nxt[c] = load_chunk(dn, c);
            }
        }
        prev_lse = lse;
        prev_valid = valid;
    }
    __syncthreads();
    if (tid == 0 && nr > 0) finish_row(row_of(nr - 1), (nr - 1) & 1, prev_lse, prev_valid);
    float* prow = ws.part + (int64_t)blockIdx.x * V;
#pragma unroll
    for (int c = 0; c < NCH; ++c) store_f32_chunk<VEC>(prow, (c * THREADS + tid) * VEC, V, &acc[c * VEC]);
    if (tid == 0) {
        ws.wg_count[blockIdx.x] = cnt;
        ws.wg_loss[blockIdx.x] = ce;
        ws.wg_flags[blockIdx.x] = bad ? BOM_FLAG_LABEL_RANGE : 0;
    }
}

// ---------------------------------------------------------------------------------------------
// Single pass, rows too wide for one workgroup (bf16): S workgroups share each row, part q owning
// columns [q W, min(V, (q + 1) W)), and together stream Z once. A part's slice of a row goes straight
// from memory into one of two LDS row buffers (buffer loads that write LDS: the slice holds no registers
// on its way), the slice of the row after next is requested as soon as a row's residual is written, and
// a single wait on the vector memory counter (which retires in issue order) tells a wave that its own
// chunks of the next row have landed; each thread reads only the slots its own wave loaded, so no
// barrier guards the buffers. Pass one keeps exp(z - m) of the thread's columns in registers (m: the
// thread's maximum), so pass two scales them by exp(m - lse) instead of evaluating exp again. Each part
// reduces its (max, sum of exp(z - max), first argmax) and publishes them as three 64-bit words
// (validity marker in the high half, value in the low half; the area is zeroed before the launch) with
// relaxed device-scope atomic stores; lane q of wave 0 then polls part q's words with relaxed
// device-scope atomic loads, and every thread combines all S records in part order, so every part
// derives the same lse. A poll is bounded: after spin_limit polls (or at once when spin_limit < 0) the
// whole workgroup reduces the missing part's slice from Z itself with the same operations in the same
// order that part runs (so the record has the same bits as the one it would have published) and stops
// waiting for that part, so the kernel finishes whatever the scheduling and its results do not depend on
// it; the flags word then carries BOM_FLAG_RESIDUAL_RECOMPUTED. The part holding a row's label (part 0
// for ignored rows) writes that row's outputs and loss term. Workgroup (g, q) writes columns of partial
// row g; the S parts of group g together fill it. Logit loads and residual stores carry the non-temporal
// hint.
template <int THREADS, int NCH>
__global__ __launch_bounds__(THREADS) void residual_split_kernel(
    const uint16_t* __restrict__ Z, int64_t ldz, int N, int V, const int32_t* __restrict__ labels, int32_t ignore_index,
    float* __restrict__ row_lse, int32_t* __restrict__ row_argmax, float* __restrict__ row_target,
    uint16_t* __restrict__ R, int64_t ldr, int S, int W, int spin_limit, Partials ws) {
    static_assert(NCH >= 2 && NCH <= kSplitMaxNch, "two LDS row buffers of NCH chunks per thread");
    constexpr int VEC = 8;
    constexpr int NW = THREADS / kWave;
    constexpr int VPT = NCH * VEC;
    __shared__ uint4 slots[2][NCH * THREADS];
    __shared__ float sh_m[2][NW];
    __shared__ float sh_l[2][NW];
    __shared__ int sh_am;
    __shared__ float sh_zt[2];
    __shared__ float sh_rec_m[kSplitMaxParts], sh_rec_l[kSplitMaxParts];   // the row's per-part records
    __shared__ int sh_rec_a[kSplitMaxParts];
    __shared__ int sh_miss;   // parts whose record did not arrive (bit q)
    __shared__ float sh_fm[NW], sh_fl[NW];   // reduction of a partner's slice
    __shared__ int sh_fam;
    const int tid = threadIdx.x;
    const int part = blockIdx.x % S, g = blockIdx.x / S, G = gridDim.x / S;
    const int c0 = part * W;
    const int Vp = min(W, V - c0);
    float acc[VPT];
#pragma unroll
    for (int k = 0; k < VPT; ++k) acc[k] = 0.f;
    const int nr = g < N ? (N - 1 - g) / G + 1 : 0;
    auto row_of = [&](int j) { return g + j * G; };
    int cnt = 0;
    double ce = 0.0;
    bool bad = false;
    bool dead = false;   // wave 0, lane q: part q is no longer waited for
    bool recomputed = false;   // some partner record was recomputed from Z (reported in the flags word)
    auto unpack = [](const uint4& u, float* x) {
        x[0] = bf16_lo(u.x); x[1] = bf16_hi(u.x); x[2] = bf16_lo(u.y); x[3] = bf16_hi(u.y);
        x[4] = bf16_lo(u.z); x[5] = bf16_hi(u.z); x[6] = bf16_lo(u.w); x[7] = bf16_hi(u.w);
    };
    const int voff = tid * 16;
    // the first chunk index of this wave's lanes whose chunks may lie past the slice's end
    const int wave_last = (tid | (kWave - 1));
    // chunk c of the thread with the columns past the end of a slice of nq columns read as -inf
    auto pad = [&](int c, int nq, uint4 w) {
        if ((c * THREADS + wave_last) * VEC >= nq) {   // uniform per wave
            const bool ok = ((c * THREADS + tid) * VEC) < nq;
            const uint32_t mk = lane_mask(ok), fb = 0xFF80FF80u & ~mk;
            w = make_uint4((w.x & mk) | fb, (w.y & mk) | fb, (w.z & mk) | fb, (w.w & mk) | fb);
        }
        return w;
    };
    // Row i's slice into LDS buffer buf: chunk c of the thread at slots[buf][c * THREADS + tid]. m0 holds the
    // LDS address of the wave's 64 slots of the chunk (each lane's 16 bytes land at m0 + 16 lane) and is
    // restored afterwards; one wait state separates the write of m0 from the load that reads it. The whole
    // byte offset goes in the VGPR operand (the scalar offset is outside the descriptor's range check), so
    // bytes past the slice's end read as zeros and nothing past it is touched; they are padded as they are
    // unpacked.
    auto issue_row = [&](int buf, int i) {
        const uint64_t pa = reinterpret_cast<uint64_t>(Z + (int64_t)i * ldz + c0);
        const i32x4_t rs = {__builtin_amdgcn_readfirstlane((int)(uint32_t)pa),
                            __builtin_amdgcn_readfirstlane((int)((uint32_t)(pa >> 32) & 0xFFFFu)),
                            __builtin_amdgcn_readfirstlane(Vp * 2), kBufFlags};
        const uint32_t lds0 = __builtin_amdgcn_readfirstlane(
            (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)(&slots[buf][tid & ~(kWave - 1)]));
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            int m0_saved;
            asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\t"
                         "buffer_load_dwordx4 %2, %3, 0 offen nt lds\n\ts_mov_b32 m0, %0"
                         : "=&s"(m0_saved)
                         : "s"(lds0 + c * THREADS * 16), "v"(voff + c * THREADS * 16), "s"(rs)
                         : "memory");
        }
    };
    // this wave's chunks of the row in the buffer about to be read have landed once at most `younger`
    // vector memory operations issued after them remain
    auto wait_landed = [](int younger) {
        if (younger >= 2 * NCH) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * NCH) : "memory");
        else if (younger >= NCH) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(NCH) : "memory");
        else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    };
    if (nr > 0) issue_row(0, row_of(0));
    if (nr > 1) issue_row(1, row_of(1));
    if (tid == 0) {
        sh_am = INT_MAX;
        sh_fam = INT_MAX;
    }
    constexpr unsigned long long kValid = 1ull << 32;
    auto xword = [&](int i, int q, int f) { return ws.xch + ((int64_t)i * S + q) * 3 + f; };
    // wave 0, lane q: part q's record of row i from its words; false when the poll bound runs out (from
    // then on part q is not waited for) or when spin_limit < 0
    auto fetch = [&](int i, int q, float* mq, float* lq, int* aq) {
        if (dead) return false;
        // the three words are polled together (one round trip per poll when the record is there)
        unsigned long long v[3];
        bool ok = false;
        for (int it = 0; spin_limit >= 0 && it <= spin_limit; ++it) {
#pragma unroll
            for (int f = 0; f < 3; ++f) v[f] = __hip_atomic_load(xword(i, q, f), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if ((v[0] >> 32) == 1 && (v[1] >> 32) == 1 && (v[2] >> 32) == 1) {
                ok = true;
                break;
            }
            __builtin_amdgcn_s_sleep(2);
        }
        if (!ok) {
            dead = true;
            return false;
        }
        *mq = __uint_as_float((uint32_t)v[0]);
        *lq = __uint_as_float((uint32_t)v[1]);
        *aq = (int)(uint32_t)v[2];
        return true;
    };
    // The reduction of one part's slice, shared by a part's own pass and by the recomputation of a
    // partner's record when that record does not arrive: the thread's maximum m over its columns (chunk
    // maxima in chunk order; cmax = the chunk where it first appears), then l = the sum, in chunk order, of
    // each chunk's pairwise sum of exp(z - m). Both callers run these same operations in the same order
    // (contraction off, explicit fma only) on the same padded chunks, so a recomputed record has the
    // partner's bits and every part derives the same lse whichever way it obtained a record.
    auto chunk_max = [](const float* x) {
        auto mx = [](float a, float b2) { return __builtin_elementwise_maximum(a, b2); };
        return mx(mx(mx(x[0], x[1]), mx(x[2], x[3])), mx(mx(x[4], x[5]), mx(x[6], x[7])));
    };
    auto max_step = [](int c, float cm, float* m, int* cmax) {
        if (c > 0 && cm > *m) *cmax = c;
        *m = __builtin_elementwise_maximum(*m, cm);
    };
    // exp(z - m) of one chunk in place (m2 = m log2 e) and its pairwise sum
    auto chunk_exp_sum = [](float* x, float m2) {
#pragma clang fp contract(off)
#pragma unroll
        for (int k = 0; k < VEC; ++k) x[k] = exp2_fast(fmaf(x[k], kLog2e, -m2));
        return ((x[0] + x[1]) + (x[2] + x[3])) + ((x[4] + x[5]) + (x[6] + x[7]));
    };
    // this part's own slice from LDS buffer b; e receives exp(z - m) of every column the thread holds
    auto own_stats = [&](int b, float* e, float* m_out, float* l_out, int* cmax_out) {
#pragma clang fp contract(off)
        float m = -INFINITY, l = 0.f;
        int cmax = 0;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            unpack(pad(c, Vp, slots[b][c * THREADS + tid]), &e[c * VEC]);
            max_step(c, chunk_max(&e[c * VEC]), &m, &cmax);
        }
        const float m2 = m * kLog2e;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const float cl = chunk_exp_sum(&e[c * VEC], m2);
            l = c == 0 ? cl : l + cl;
        }
        *m_out = m;
        *l_out = l;
        *cmax_out = cmax;
    };
    // a partner's slice, chunk_at(c) loading this thread's padded chunk c of it (read once per sweep; the
    // loops stay rolled, so that this rare path holds one chunk at a time and adds no register pressure to
    // the rest of the kernel)
    auto partner_stats = [&](auto&& chunk_at, float* m_out, float* l_out, int* cmax_out) {
#pragma clang fp contract(off)
        float m = -INFINITY, l = 0.f;
        int cmax = 0;
#pragma unroll 1
        for (int c = 0; c < NCH; ++c) {
            float x[VEC];
            unpack(chunk_at(c), x);
            max_step(c, chunk_max(x), &m, &cmax);
        }
        const float m2 = m * kLog2e;
#pragma unroll 1
        for (int c = 0; c < NCH; ++c) {
            float x[VEC];
            unpack(chunk_at(c), x);
            const float cl = chunk_exp_sum(x, m2);
            l = c == 0 ? cl : l + cl;
        }
        *m_out = m;
        *l_out = l;
        *cmax_out = cmax;
    };
    // wave reduction of (m, l) into shm[wave], shl[wave] (the caller then passes a barrier); DPP lane
    // permutes, so the chain of steps makes no LDS round trips
    auto wave_stats = [&](float m, float l, float* shm, float* shl) {
#pragma clang fp contract(off)
        const float mw = wave_max_dpp(m);
        const float lw = wave_sum_dpp(l * exp2_fast((m - mw) * kLog2e));
        if ((tid & (kWave - 1)) == 0) {
            shm[tid / kWave] = mw;
            shl[tid / kWave] = lw;
        }
    };
    // the workgroup's (max, sum) from the per-wave values (uniform): lanes 0 .. NW - 1 of every wave hold
    // them, so one 16-lane row reduces them
    static_assert(NW <= 16, "the per-wave values fit one 16-lane row");
    auto group_stats = [&](const float* shm, const float* shl, float* mp, float* lp) {
#pragma clang fp contract(off)
        const int lane = tid & (kWave - 1);
        const float mg = lane < NW ? shm[lane] : -INFINITY;
        const float mm = lane_f32(row16_max(mg), 0);
        const float lg = lane < NW ? shl[lane] * exp2_fast((mg - mm) * kLog2e) : 0.f;
        *mp = mm;
        *lp = lane_f32(row16_sum(lg), 0);
    };
    // first column of chunk cmax holding the maximum mp (the lowest one over the workgroup, by atomicMin)
    auto first_max = [&](const uint4& w, int cmax, float mp, int* sh) {
        float x[VEC];
        unpack(w, x);
        int k0 = VEC - 1;
#pragma unroll
        for (int k = VEC - 2; k >= 0; --k) k0 = (x[k] == mp) ? k : k0;
        atomicMin(sh, (cmax * THREADS + tid) * VEC + k0);
    };
    auto finish_row = [&](int i, int b, float lse, bool valid, int am) {
        if (row_argmax) row_argmax[i] = am;
        const float zt = valid ? sh_zt[b] : 0.f;
        if (row_target) row_target[i] = zt;
        row_lse[i] = lse;
        if (valid) {
            ++cnt;
            ce += (double)lse - (double)zt;
        }
    };
    float prev_lse = 0.f;
    bool prev_valid = false, prev_own = false;
    int prev_am = 0;
    for (int j = 0; j < nr; ++j) {
        const int i = row_of(j);
        const int b = j & 1;
        // vector memory operations this wave issued after row j's loads: row j - 1's residual stores, then
        // row j + 1's loads
        wait_landed((j > 0 ? NCH : 0) + (j + 1 < nr ? NCH : 0));
        // pass 1 (LDS): (max, sum of exp(z - max)) of this thread's columns; their exp(z - max) stay in e
        float e[VPT];
        float m_thread, l;
        int cmax;
        own_stats(b, e, &m_thread, &l, &cmax);
        wave_stats(m_thread, l, sh_m[b], sh_l[b]);
        __syncthreads();
        if (tid == 0 && j > 0 && prev_own) finish_row(row_of(j - 1), b ^ 1, prev_lse, prev_valid, prev_am);
        float mp, lp;
        group_stats(sh_m[b], sh_l[b], &mp, &lp);
        if (m_thread == mp) first_max(pad(cmax, Vp, slots[b][cmax * THREADS + tid]), cmax, mp, &sh_am);
        __syncthreads();
        // wave 0: lane 0 publishes this part's record; lane q < S fetches part q's (all in parallel)
        if (tid < kWave) {
            const int ap = c0 + sh_am;
            if (tid == 0) {
                sh_am = INT_MAX;   // next written after the next row's first barrier
                __hip_atomic_store(xword(i, part, 0), kValid | __float_as_uint(mp), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(xword(i, part, 1), kValid | __float_as_uint(lp), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(xword(i, part, 2), kValid | (uint32_t)ap, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            }
            float mq = mp, lq = lp;
            int aq = ap;
            bool have = true;
            if (tid < S && tid != part) have = fetch(i, tid, &mq, &lq, &aq);
            if (tid < S) {
                sh_rec_m[tid] = mq;
                sh_rec_l[tid] = lq;
                sh_rec_a[tid] = aq;
            }
            const unsigned long long miss = __ballot(tid < S && !have);
            if (tid == 0) sh_miss = (int)(miss & ((1u << kSplitMaxParts) - 1));
        }
        __syncthreads();
        // records that did not arrive: the whole workgroup reduces that part's slice from Z
        const int missing = sh_miss;
        if (missing != 0) recomputed = true;
        for (int miss = missing; miss != 0; miss &= miss - 1) {
            const int q = __builtin_ctz(miss);
            const int q0 = q * W, nq = min(W, V - q0);
            const auto dq = make_desc(Z + (int64_t)i * ldz + q0, nq * 2);
            auto chunk_q = [&](int c) {
                const u32x4_t w = __builtin_amdgcn_raw_buffer_load_b128(dq, voff + c * THREADS * 16, 0, kNonTemporal);
                return pad(c, nq, make_uint4(w[0], w[1], w[2], w[3]));
            };
            float mt, lt, mq, lq;
            int cq;
            partner_stats(chunk_q, &mt, &lt, &cq);
            wave_stats(mt, lt, sh_fm, sh_fl);
            __syncthreads();
            group_stats(sh_fm, sh_fl, &mq, &lq);
            if (mt == mq) first_max(chunk_q(cq), cq, mq, &sh_fam);
            __syncthreads();
            if (tid == 0) {
                sh_rec_m[q] = mq;
                sh_rec_l[q] = lq;
                sh_rec_a[q] = q0 + sh_fam;
                sh_fam = INT_MAX;
            }
            __syncthreads();
        }
        // the recomputation reused the registers of e: rebuild it from the slots (the same values)
        if (missing != 0) own_stats(b, e, &m_thread, &l, &cmax);
        // every thread combines the S records in part order (the same operations in every part)
        float M = -INFINITY, L = 0.f;
        int A = 0;
        {
#pragma clang fp contract(off)
            for (int q = 0; q < S; ++q) {
                const float m2 = sh_rec_m[q], l2 = sh_rec_l[q];
                const int a2 = sh_rec_a[q];
                if (q == 0) {
                    M = m2;
                    L = l2;
                    A = a2;
                } else if (m2 > M) {
                    L = fmaf(L, exp2_fast((M - m2) * kLog2e), l2);
                    M = m2;
                    A = a2;
                } else {
                    L = fmaf(l2, exp2_fast((m2 - M) * kLog2e), L);
                }
            }
        }
        const float lse = M + logf(L);
        const int y = labels[i];
        bool rbad = false;
        const bool valid = label_valid(y, V, ignore_index, &rbad);
        const bool own = valid ? (y / W == part) : (part == 0);
        if (own) bad |= rbad;
        const auto rdesc = make_desc(R ? R + (int64_t)i * ldr + c0 : nullptr, R ? Vp * 2 : 0);
        const int yl = y - c0;
        const bool here = valid && yl >= 0 && yl < Vp;
        const int yv = yl / VEC;
        const int slot = (here && yv % THREADS == tid) ? (yv / THREADS) * VEC + (yl % VEC) : -1;
        // pass 2 (registers): p = exp(z - lse) = exp(z - m) exp(m - lse), one scale per thread
        const float sc = exp2_fast(m_thread * kLog2e - lse * kLog2e);
        if (slot >= 0) {
            const uint32_t w = reinterpret_cast<const uint32_t*>(&slots[b][(slot / VEC) * THREADS + tid])[(slot % VEC) >> 1];
            sh_zt[b] = (slot & 1) ? bf16_hi(w) : bf16_lo(w);
        }
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            float p[VEC];
            if (valid) {
#pragma unroll
                for (int k = 0; k < VEC; ++k) p[k] = e[c * VEC + k] * sc;
                if (slot >= 0) {
#pragma unroll
                    for (int k = 0; k < VEC; ++k)
                        if (c * VEC + k == slot) p[k] -= 1.0f;
                }
#pragma unroll
                for (int k = 0; k < VEC; ++k) acc[c * VEC + k] += p[k];
            } else {
#pragma unroll
                for (int k = 0; k < VEC; ++k) p[k] = 0.f;
            }
            u32x4_t w;
            w[0] = pack_bf16x2(p[0], p[1]);
            w[1] = pack_bf16x2(p[2], p[3]);
            w[2] = pack_bf16x2(p[4], p[5]);
            w[3] = pack_bf16x2(p[6], p[7]);
            __builtin_amdgcn_raw_buffer_store_b128(w, rdesc, voff + c * THREADS * 16, 0, kNonTemporal);
        }
        // buffer b is free once this thread's reads of it are done (its own wave loaded every slot it reads)
        if (j + 2 < nr) issue_row(b, row_of(j + 2));
        prev_lse = lse;
        prev_valid = valid;
        prev_own = own;
        prev_am = A;
    }
    __syncthreads();
    if (tid == 0 && nr > 0 && prev_own) finish_row(row_of(nr - 1), (nr - 1) & 1, prev_lse, prev_valid, prev_am);
    float* prow = ws.part + (int64_t)g * V + c0;
#pragma unroll
    for (int c = 0; c < NCH; ++c) store_f32_chunk<VEC>(prow, (c * THREADS + tid) * VEC, Vp, &acc[c * VEC]);
    if (tid == 0) {
        ws.wg_count[blockIdx.x] = cnt;
        ws.wg_loss[blockIdx.x] = ce;
        ws.wg_flags[blockIdx.x] = (bad ? BOM_FLAG_LABEL_RANGE : 0) | (recomputed ? BOM_FLAG_RESIDUAL_RECOMPUTED : 0);
    }
}

__global__ void zero_u64_kernel(unsigned long long* __restrict__ p, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0ull;
}

// ---------------------------------------------------------------------------------------------
// Two pass, stats: one wave per row, online (max, sum, argmax) per lane, then a butterfly merge.
template <typename T, int VEC, int UNROLL>
__global__ __launch_bounds__(kStatsRowsPerWG * kWave) void residual_stats_kernel(
    const T* __restrict__ Z, int64_t ldz, int N, int V, const int32_t* __restrict__ labels, int32_t ignore_index,
    float* __restrict__ row_lse, int32_t* __restrict__ row_argmax, float* __restrict__ row_target, Partials ws) {
    constexpr int STEP = kWave * VEC * UNROLL;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int i = blockIdx.x * kStatsRowsPerWG + wave;
    float m = -INFINITY, l = 0.f;
    int idx = INT_MAX;
    if (i < N) {
        const T* zr = Z + (int64_t)i * ldz;
        for (int base = 0; base < V; base += STEP) {
            float x[UNROLL * VEC];
#pragma unroll
            for (int u = 0; u < UNROLL; ++u) load_chunk<T, VEC>(zr, base + (u * kWave + lane) * VEC, V, -INFINITY, &x[u * VEC]);
            float cm = -INFINITY;
#pragma unroll
            for (int k = 0; k < UNROLL * VEC; ++k) cm = fmaxf(cm, x[k]);
            if (cm > m) {
                int ci = INT_MAX;
#pragma unroll
                for (int u = UNROLL - 1; u >= 0; --u)
#pragma unroll
                    for (int k = VEC - 1; k >= 0; --k)
                        if (x[u * VEC + k] == cm) ci = base + (u * kWave + lane) * VEC + k;
                l = (m == -INFINITY) ? 0.f : l * exp2_fast((m - cm) * kLog2e);
                m = cm;
                idx = ci;
            }
            if (m != -INFINITY) {  // a lane that has only seen padding keeps l = 0
                const float m2 = m * kLog2e;
#pragma unroll
                for (int k = 0; k < UNROLL * VEC; ++k) l += exp2_fast(fmaf(x[k], kLog2e, -m2));
            }
        }
    }
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) {
        const float mo = __shfl_xor(m, o, kWave);
        const float lo = __shfl_xor(l, o, kWave);
        const int io = __shfl_xor(idx, o, kWave);
        const float mn = fmaxf(m, mo);
        const float a = (m == -INFINITY) ? 0.f : l * exp2_fast((m - mn) * kLog2e);
        const float b = (mo == -INFINITY) ? 0.f : lo * exp2_fast((mo - mn) * kLog2e);
        l = a + b;
        idx = (m > mo) ? idx : (mo > m ? io : min(idx, io));
        m = mn;
    }
    __shared__ int sh_cnt[kStatsRowsPerWG];
    __shared__ int sh_bad[kStatsRowsPerWG];
    __shared__ double sh_ce[kStatsRowsPerWG];
    if (lane == 0) {
        int c = 0, bd = 0;
        double e = 0.0;
        if (i < N) {
            const float lse = m + logf(l);
            const int y = labels[i];
            bool rbad = false;
            const bool valid = label_valid(y, V, ignore_index, &rbad);
            const float zt = valid ? load_scalar<T>(Z + (int64_t)i * ldz + y) : 0.f;
            row_lse[i] = lse;
            if (row_argmax) row_argmax[i] = idx;
            if (row_target) row_target[i] = zt;
            c = valid ? 1 : 0;
            bd = rbad ? 1 : 0;
            e = valid ? (double)lse - (double)zt : 0.0;
        }
        sh_cnt[wave] = c;
        sh_bad[wave] = bd;
        sh_ce[wave] = e;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int c = 0, bd = 0;
        double e = 0.0;
        for (int w = 0; w < kStatsRowsPerWG; ++w) {
            c += sh_cnt[w];
            bd |= sh_bad[w];
            e += sh_ce[w];
        }
        ws.wg_count[blockIdx.x] = c;
        ws.wg_loss[blockIdx.x] = e;
        ws.wg_flags[blockIdx.x] = bd ? BOM_FLAG_LABEL_RANGE : 0;
    }
}

// Two pass, columns: workgroup (cb, rb) owns columns col0 + (c * THREADS + tid) * VEC + k and rows
// [rb * row_block, ...); p = exp(z - lse) with the stats kernel's lse.
template <typename T, int VEC>
__global__ __launch_bounds__(kColsThreads) void residual_cols_kernel(
    const T* __restrict__ Z, int64_t ldz, int N, int V, const int32_t* __restrict__ labels, int32_t ignore_index,
    const float* __restrict__ row_lse, T* __restrict__ R, int64_t ldr, int row_block, float* __restrict__ part) {
    constexpr int VPT = kColsCPT * VEC;
    constexpr int SLAB = kColsThreads * VPT;
    const int tid = threadIdx.x;
    const int nslab = (V + SLAB - 1) / SLAB;
    const int cb = blockIdx.x % nslab, rb = blockIdx.x / nslab;
    const int col0 = cb * SLAB;
    const int r0 = rb * row_block;
    const int r1 = min(N, r0 + row_block);
    float acc[VPT];
#pragma unroll
    for (int k = 0; k < VPT; ++k) acc[k] = 0.f;
    for (int i = r0; i < r1; ++i) {
        const int y = labels[i];
        bool rbad = false;
        const bool valid = label_valid(y, V, ignore_index, &rbad);
        T* rr = R ? R + (int64_t)i * ldr : nullptr;
        if (!valid) {
            if (rr) {
                float zero[VEC];
#pragma unroll
                for (int k = 0; k < VEC; ++k) zero[k] = 0.f;
#pragma unroll
                for (int c = 0; c < kColsCPT; ++c) store_chunk<T, VEC>(rr, col0 + (c * kColsThreads + tid) * VEC, V, zero);
            }
            continue;
        }
        const T* zr = Z + (int64_t)i * ldz;
        const float lse2 = row_lse[i] * kLog2e;
        float x[VPT];
#pragma unroll
        for (int c = 0; c < kColsCPT; ++c) load_chunk<T, VEC>(zr, col0 + (c * kColsThreads + tid) * VEC, V, -INFINITY, &x[c * VEC]);
#pragma unroll
        for (int k = 0; k < VPT; ++k) x[k] = exp2_fast(fmaf(x[k], kLog2e, -lse2));
        const int yl = y - col0;
        if (yl >= 0 && yl < SLAB && (yl / VEC) % kColsThreads == tid) {
            const int slot = ((yl / VEC) / kColsThreads) * VEC + (yl % VEC);
#pragma unroll
            for (int k = 0; k < VPT; ++k)
                if (k == slot) x[k] -= 1.0f;
        }
#pragma unroll
        for (int k = 0; k < VPT; ++k) acc[k] += x[k];
        if (rr) {
#pragma unroll
            for (int c = 0; c < kColsCPT; ++c) store_chunk<T, VEC>(rr, col0 + (c * kColsThreads + tid) * VEC, V, &x[c * VEC]);
        }
    }
    float* prow = part + (int64_t)rb * V;
#pragma unroll
    for (int c = 0; c < kColsCPT; ++c) store_f32_chunk<VEC>(prow, col0 + (c * kColsThreads + tid) * VEC, V, &acc[c * VEC]);
}

// ---------------------------------------------------------------------------------------------
// Finish: s_j = (sum of the partial column sums, in a fixed order) / N_t. Workgroup b owns columns
// b*64 .. b*64+63 (one per lane); wave w adds partials w, w+16, ... and the 16 wave sums are added
// in wave order. Every workgroup sums the per-workgroup row counts itself (integers: exact in any
// order) to get N_t; workgroup 0 also writes N_t, the flags and the loss (fp64 sum, fixed order).
constexpr int kFinThreads = 1024;
constexpr int kFinWaves = kFinThreads / kWave;

__global__ __launch_bounds__(kFinThreads) void residual_finish_kernel(int nparts, int V, int nwg, Partials ws,
                                                                      float* __restrict__ s, float* __restrict__ loss,
                                                                      int32_t* __restrict__ n_valid,
                                                                      int32_t* __restrict__ flags) {
    __shared__ float sh_s[kFinWaves][kWave];
    __shared__ int sh_c[kFinWaves];
    __shared__ int sh_f[kFinWaves];
    __shared__ double sh_l[kFinWaves];
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int j = blockIdx.x * kWave + lane;
    const int jc = j < V ? j : V - 1;
    const float* __restrict__ part = ws.part;
    float a = 0.f;
    int p = wave;
    for (; p + 3 * kFinWaves < nparts; p += 4 * kFinWaves) {
        const float p0 = part[(int64_t)p * V + jc];
        const float p1 = part[(int64_t)(p + kFinWaves) * V + jc];
        const float p2 = part[(int64_t)(p + 2 * kFinWaves) * V + jc];
        const float p3 = part[(int64_t)(p + 3 * kFinWaves) * V + jc];
        a += p0;
        a += p1;
        a += p2;
        a += p3;
    }
    for (; p < nparts; p += kFinWaves) a += part[(int64_t)p * V + jc];
    sh_s[wave][lane] = a;
    int c = 0;
    for (int w = threadIdx.x; w < nwg; w += kFinThreads) c += ws.wg_count[w];
    c = wave_sum(c);
    if (lane == 0) sh_c[wave] = c;
    const bool first = blockIdx.x == 0;
    if (first) {
        int f = 0;
        double e = 0.0;
        for (int w = threadIdx.x; w < nwg; w += kFinThreads) {
            f |= ws.wg_flags[w];
            e += ws.wg_loss[w];
        }
        f = wave_or(f);
        e = wave_sum(e);
        if (lane == 0) {
            sh_f[wave] = f;
            sh_l[wave] = e;
        }
    }
    __syncthreads();
    if (wave != 0) return;
    int nt = 0;
#pragma unroll
    for (int w = 0; w < kFinWaves; ++w) nt += sh_c[w];
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < kFinWaves; ++w) sum += sh_s[w][lane];
    const float inv_nt = nt > 0 ? (float)(1.0 / (double)nt) : 0.f;
    if (j < V) s[j] = sum * inv_nt;
    if (first && lane == 0) {
        int f = 0;
        double e = 0.0;
        for (int w = 0; w < kFinWaves; ++w) {
            f |= sh_f[w];
            e += sh_l[w];
        }
        *n_valid = nt;
        *flags = f | (nt == 0 ? BOM_FLAG_EMPTY : 0);
        *loss = nt > 0 ? (float)(e / (double)nt) : 0.f;
    }
}

// ---------------------------------------------------------------------------------------------
template <int THREADS, int NCH>
hipError_t launch_rows_lds(const uint16_t* Z, int64_t ldz, int N, int V, const int32_t* labels, int32_t ignore_index,
                           float* row_lse, int32_t* row_argmax, float* row_target, uint16_t* R, int64_t ldr, Partials ws,
                           int* nwg_out, hipStream_t stream) {
    int nwg = N < kSingleMaxWG ? N : kSingleMaxWG;
    const int rpw = (N + nwg - 1) / nwg;
    nwg = (N + rpw - 1) / rpw;
    *nwg_out = nwg;
    hipLaunchKernelGGL((residual_rows_lds_kernel<THREADS, NCH>), dim3(nwg), dim3(THREADS), 0, stream, Z, ldz, N, V, labels,
                       ignore_index, row_lse, row_argmax, row_target, R, ldr, rpw, ws);
    return hipGetLastError();
}

template <typename T, int THREADS, int VEC, int NCH>
hipError_t launch_rows(const T* Z, int64_t ldz, int N, int V, const int32_t* labels, int32_t ignore_index, float* row_lse,
                       int32_t* row_argmax, float* row_target, T* R, int64_t ldr, Partials ws, int* nwg_out,
                       hipStream_t stream) {
    int nwg = N < kSingleMaxWG ? N : kSingleMaxWG;
    const int rpw = (N + nwg - 1) / nwg;
    nwg = (N + rpw - 1) / rpw;
    *nwg_out = nwg;
    // wide bf16 rows at 512 threads keep raw pairs (registers: acc + packed row) instead of fp32 e
    constexpr bool kPacked = (VEC == 8) && (NCH > 8);
    hipLaunchKernelGGL((residual_rows_kernel<T, THREADS, VEC, NCH, kPacked>), dim3(nwg), dim3(THREADS), 0, stream, Z,
                       ldz, N, V, labels, ignore_index, row_lse, row_argmax, row_target, R, ldr, rpw, ws);
    return hipGetLastError();
}

// Allowed chunk counts for 512-thread single-pass workgroups (registers: 2 * NCH * VEC floats).
constexpr int kNchSet[] = {1, 2, 3, 4, 6, 8, 10, 13};
constexpr int kLdsNchSet[] = {2, 3, 4, 6, 8, 10, 12, 13, 14};
constexpr int kLds1kNchSet[] = {2, 3, 4, 5, 6};

template <typename T, int VEC>
hipError_t dispatch_rows(int nch, int threads, const T* Z, int64_t ldz, int N, int V, const int32_t* labels,
                         int32_t ig, float* lse, int32_t* am, float* tg, T* R, int64_t ldr, Partials ws, int* nwg,
                         hipStream_t st) {
#define BOM_ROWS(TH, NC) launch_rows<T, TH, VEC, NC>(Z, ldz, N, V, labels, ig, lse, am, tg, R, ldr, ws, nwg, st)
    if (threads == 64) return BOM_ROWS(64, 1);
    if (threads == 128) return BOM_ROWS(128, 1);
    if (threads == 256) return BOM_ROWS(256, 1);
    if (threads == 1024) {
        switch (nch) {
            case 1: return BOM_ROWS(1024, 1);
            case 2: return BOM_ROWS(1024, 2);
            case 3: return BOM_ROWS(1024, 3);
            case 4: return BOM_ROWS(1024, 4);
            default: return hipErrorInvalidValue;
        }
    }
    if constexpr (std::is_same<T, uint16_t>::value && VEC == 8) {
        if (threads == -512) {   // bf16 rows parked in LDS, next row prefetched
#define BOM_LDS(NC) launch_rows_lds<512, NC>(Z, ldz, N, V, labels, ig, lse, am, tg, R, ldr, ws, nwg, st)
            switch (nch) {
                case 2: return BOM_LDS(2);
                case 3: return BOM_LDS(3);
                case 4: return BOM_LDS(4);
                case 6: return BOM_LDS(6);
                case 8: return BOM_LDS(8);
                case 10: return BOM_LDS(10);
                case 12: return BOM_LDS(12);
                case 13: return BOM_LDS(13);
                case 14: return BOM_LDS(14);
                default: return hipErrorInvalidValue;
            }
#undef BOM_LDS
        }
        if (threads == -1024) {   // the same with 1024-thread workgroups (16 waves per CU)
#define BOM_LDS(NC) launch_rows_lds<1024, NC>(Z, ldz, N, V, labels, ig, lse, am, tg, R, ldr, ws, nwg, st)
            switch (nch) {
                case 2: return BOM_LDS(2);
                case 3: return BOM_LDS(3);
                case 4: return BOM_LDS(4);
                case 5: return BOM_LDS(5);
                case 6: return BOM_LDS(6);
                default: return hipErrorInvalidValue;
            }
#undef BOM_LDS
        }
    }
    switch (nch) {
        case 1: return BOM_ROWS(512, 1);
        case 2: return BOM_ROWS(512, 2);
        case 3: return BOM_ROWS(512, 3);
        case 4: return BOM_ROWS(512, 4);
        case 6: return BOM_ROWS(512, 6);
        case 8: return BOM_ROWS(512, 8);
        case 10: return BOM_ROWS(512, 10);
        case 13: return BOM_ROWS(512, 13);
        default: return hipErrorInvalidValue;
    }
#undef BOM_ROWS
}

// Variant override for A/B measurement (environment BOM_RESIDUAL_PLAN, read once):
// 0 automatic, 1 = 512-thread register rows, 2 = 1024-thread register rows, 3 = two pass,
// 4 = 1024-thread LDS rows where they fit, 5 = 512-thread LDS rows, 6 = split rows (at least two
// parts) for every bf16 row wider than one workgroup's 512 threads.
int plan_override() {
    static const int v = [] {
        const char* e = getenv("BOM_RESIDUAL_PLAN");
        return e ? atoi(e) : 0;
    }();
    return v;
}

// Single-pass plan for VEC-wide chunks: returns false when a row does not fit in registers.
// Wide rows use 1024-thread workgroups (16 waves per CU): up to 4 chunks keep fp32 e values in
// registers, 5..7 chunks (bf16 only) park the raw row in LDS.
bool plan_single(int V, int VEC, int* threads, int* nch) {
    const int ov = plan_override();
    if (ov == 3 || ov == 6) return false;
    const int slots = (V + VEC - 1) / VEC;
    int th = 64;
    while (th < slots && th < 512) th *= 2;
    const int need = (slots + th - 1) / th;
    if (th < 512) {
        *threads = th;
        *nch = 1;
        return true;
    }
    const int need1k = (slots + 1023) / 1024;
    // automatic: bf16 rows of 2..6 chunks per thread at 1024 threads are parked in LDS by
    // 1024-thread workgroups (16 waves per CU hide more latency), wider ones by 512-thread
    // workgroups (up to 14 chunks); both prefetch the next row into registers (threads = -1024 or
    // -512 mark those kernels); fp32 rows use 512-thread register rows up to 8 chunks, then
    // 1024-thread register rows
    if (VEC == 8 && (ov == 4 || ov == 0) && need1k >= 2 && need1k <= 6) {
        for (int c : kLds1kNchSet) {
            if (c >= need1k) {
                *threads = -1024;
                *nch = c;
                return true;
            }
        }
    }
    if (VEC == 8 && (ov == 0 || ov == 5) && need >= 2) {
        for (int c : kLdsNchSet) {
            if (c >= need) {
                *threads = -512;
                *nch = c;
                return true;
            }
        }
    }
    const bool use1k = ov == 2 || (ov == 0 && need > 8);
    if (use1k && slots > 512 && need1k <= 4 && VEC != 1) {
        *threads = 1024;
        *nch = need1k;
        return true;
    }
    const int max_nch = (VEC == 1) ? 8 : 13;
    for (int c : kNchSet) {
        if (c >= need && c <= max_nch) {
            *threads = 512;
            *nch = c;
            return true;
        }
    }
    return false;
}

// Split-row plan for bf16 rows of 16-byte chunks that no single workgroup holds: S parts (at most
// kSplitMaxParts, so V up to 524,288) of at most kSplitMaxNch chunks per thread at 1024 threads; part
// width W columns (a multiple of 8). Two LDS row buffers of four chunks fill 128 KB of the CU's LDS.
bool plan_split(int V, int* S, int* W, int* nch) {
    const int slots = V / 8;
    int parts = (slots + 1024 * kSplitMaxNch - 1) / (1024 * kSplitMaxNch);
    if (plan_override() == 6 && parts < 2 && slots > 512) parts = 2;
    if (parts < 2 || parts > kSplitMaxParts) return false;
    const int per = (slots + parts - 1) / parts;
    if ((parts - 1) * per >= slots) return false;   // every part holds columns
    // every thread holds columns of every part (a thread with padding only would turn its sum into NaN);
    // the automatic plan always gives a part more than 2048 chunks, only the override can give fewer
    if (slots - (parts - 1) * per <= 1024) return false;
    *S = parts;
    *W = per * 8;
    *nch = (per + 1023) / 1024 < 2 ? 2 : (per + 1023) / 1024;
    return true;
}

// Poll bound of the split-row exchange (environment BOM_RESIDUAL_SPIN, read once; negative: never
// wait, every workgroup computes the other parts' records itself).
int split_spin_limit() {
    static const int v = [] {
        const char* e = getenv("BOM_RESIDUAL_SPIN");
        return e ? atoi(e) : (1 << 16);
    }();
    return v;
}

hipError_t launch_split(const uint16_t* Z, int64_t ldz, int N, int V, const int32_t* labels, int32_t ig, float* lse,
                        int32_t* am, float* tg, uint16_t* R, int64_t ldr, Partials ws, int S, int W, int nch, int* nwg,
                        int* nparts, hipStream_t st) {
    const int G = N < kSingleMaxWG / S ? N : kSingleMaxWG / S;
    const int64_t nx = (int64_t)N * S * 3;
    hipLaunchKernelGGL(zero_u64_kernel, dim3((unsigned)((nx + 255) / 256)), dim3(256), 0, st, ws.xch, nx);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int spin = split_spin_limit();
#define BOM_SPLIT(NC)                                                                                              \
    hipLaunchKernelGGL((residual_split_kernel<1024, NC>), dim3(S * G), dim3(1024), 0, st, Z, ldz, N, V, labels, ig, \
                       lse, am, tg, R, ldr, S, W, spin, ws)
    switch (nch) {
        case 2: BOM_SPLIT(2); break;
        case 3: BOM_SPLIT(3); break;
        case 4: BOM_SPLIT(4); break;
        default: return hipErrorInvalidValue;
    }
#undef BOM_SPLIT
    *nwg = S * G;
    *nparts = G;
    return hipGetLastError();
}

template <typename T, int VEC>
hipError_t run_residual(const T* Z, int N, int V, int64_t ldz, const int32_t* labels, int32_t ig, float* s, float* lse,
                        int32_t* am, float* tg, T* R, int64_t ldr, float* loss, int32_t* n_valid, int32_t* flags,
                        Partials ws, hipStream_t st) {
    int threads = 0, nch = 0, nwg = 0, nparts = 0;
    hipError_t e;
    int S = 0, W = 0;
    bool split = false;
    if constexpr (std::is_same<T, uint16_t>::value && VEC == 8) split = plan_split(V, &S, &W, &nch);
    if (plan_single(V, VEC, &threads, &nch)) {
        e = dispatch_rows<T, VEC>(nch, threads, Z, ldz, N, V, labels, ig, lse, am, tg, R, ldr, ws, &nwg, st);
        nparts = nwg;
    } else if (split) {
        if constexpr (std::is_same<T, uint16_t>::value && VEC == 8)
            e = launch_split(Z, ldz, N, V, labels, ig, lse, am, tg, R, ldr, ws, S, W, nch, &nwg, &nparts, st);
    } else {
        nwg = (N + kStatsRowsPerWG - 1) / kStatsRowsPerWG;
        constexpr int UNROLL = VEC == 1 ? 8 : 4;
        hipLaunchKernelGGL((residual_stats_kernel<T, VEC, UNROLL>), dim3(nwg), dim3(kStatsRowsPerWG * kWave), 0, st, Z,
                           ldz, N, V, labels, ig, lse, am, tg, ws);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        const int slab = kColsThreads * kColsCPT * VEC;
        const int rb = cols_row_block(N, V, VEC);
        nparts = (N + rb - 1) / rb;
        dim3 grid((unsigned)(((V + slab - 1) / slab) * nparts));
        hipLaunchKernelGGL((residual_cols_kernel<T, VEC>), grid, dim3(kColsThreads), 0, st, Z, ldz, N, V, labels, ig,
                           lse, R, ldr, rb, ws.part);
        e = hipGetLastError();
    }
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(residual_finish_kernel, dim3((V + kWave - 1) / kWave), dim3(kFinThreads), 0, st, nparts, V, nwg,
                       ws, s, loss, n_valid, flags);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------------------------
// Residual from the forward's row statistics: the head forward's epilogue already reduced each 256-column
// tile of every row (max, sum of exp(z - max), first argmax), so one wave per row merges the row's tile
// records in a fixed order (lane t takes tiles t, t + 64, ...; then a butterfly with the same tie rule as
// residual_stats_kernel: the lower column wins equal maxima) into lse and argmax, and forms the row's
// count and loss term with the target logit the forward wrote. The column-slab kernel then re-reads Z
// once for R and the column sums: no row is shared between workgroups, so nothing is exchanged.
__global__ __launch_bounds__(kStatsRowsPerWG * kWave) void residual_combine_kernel(
    const float* __restrict__ stats, int nT, int N, int V, const int32_t* __restrict__ labels, int32_t ignore_index,
    float* __restrict__ row_lse, int32_t* __restrict__ row_argmax, float* __restrict__ row_target, Partials ws) {
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int i = blockIdx.x * kStatsRowsPerWG + wave;
    float m = -INFINITY, l = 0.f;
    int idx = INT_MAX;
    if (i < N) {
        const float* rec = stats + (int64_t)i * nT * 3;
        for (int t = lane; t < nT; t += kWave) {
            const float mt = rec[t * 3], lt = rec[t * 3 + 1];
            const int at = __float_as_int(rec[t * 3 + 2]);
            if (mt > m) {
                l = (m == -INFINITY ? 0.f : l * exp2_fast((m - mt) * kLog2e)) + lt;
                m = mt;
                idx = at;
            } else {
                l += lt * exp2_fast((mt - m) * kLog2e);
                if (mt == m) idx = min(idx, at);
            }
        }
    }
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) {
        const float mo = __shfl_xor(m, o, kWave);
        const float lo = __shfl_xor(l, o, kWave);
        const int io = __shfl_xor(idx, o, kWave);
        const float mn = fmaxf(m, mo);
        const float a = (m == -INFINITY) ? 0.f : l * exp2_fast((m - mn) * kLog2e);
        const float b = (mo == -INFINITY) ? 0.f : lo * exp2_fast((mo - mn) * kLog2e);
        l = a + b;
        idx = (m > mo) ? idx : (mo > m ? io : min(idx, io));
        m = mn;
    }
    __shared__ int sh_cnt[kStatsRowsPerWG];
    __shared__ int sh_bad[kStatsRowsPerWG];
    __shared__ double sh_ce[kStatsRowsPerWG];
    if (lane == 0) {
        int c = 0, bd = 0;
        double e = 0.0;
        if (i < N) {
            const float lse = m + logf(l);
            bool rbad = false;
            const bool valid = label_valid(labels[i], V, ignore_index, &rbad);
            const float zt = valid ? row_target[i] : 0.f;   // the forward wrote the valid rows' targets
            row_lse[i] = lse;
            if (row_argmax) row_argmax[i] = idx;
            row_target[i] = zt;
            c = valid ? 1 : 0;
            bd = rbad ? 1 : 0;
            e = valid ? (double)lse - (double)zt : 0.0;
        }
        sh_cnt[wave] = c;
        sh_bad[wave] = bd;
        sh_ce[wave] = e;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int c = 0, bd = 0;
        double e = 0.0;
        for (int w = 0; w < kStatsRowsPerWG; ++w) {
            c += sh_cnt[w];
            bd |= sh_bad[w];
            e += sh_ce[w];
        }
        ws.wg_count[blockIdx.x] = c;
        ws.wg_loss[blockIdx.x] = e;
        ws.wg_flags[blockIdx.x] = bd ? BOM_FLAG_LABEL_RANGE : 0;
    }
}

struct StatsLayout {
    size_t stats_off, part_off, count_off, flags_off, loss_off, total;
    int nT, rb, nparts, nwg;
};

StatsLayout stats_layout(int64_t N, int64_t V) {
    StatsLayout L;
    L.nT = (int)((V + 255) / 256);
    L.rb = cols_row_block(N, V, 8);
    L.nparts = (int)((N + L.rb - 1) / L.rb);
    L.nwg = (int)((N + kStatsRowsPerWG - 1) / kStatsRowsPerWG);
    L.stats_off = 0;
    L.part_off = align256((size_t)N * L.nT * 3 * sizeof(float));
    L.count_off = align256(L.part_off + (size_t)L.nparts * V * sizeof(float));
    L.flags_off = align256(L.count_off + (size_t)L.nwg * sizeof(int));
    L.loss_off = align256(L.flags_off + (size_t)L.nwg * sizeof(int));
    L.total = align256(L.loss_off + (size_t)L.nwg * sizeof(double));
    return L;
}

}  // namespace

size_t residual_workspace_bytes(int64_t N, int64_t V, bom_dtype) { return ws_layout(N, V).total; }

hipError_t launch_residual(const void* Z, bom_dtype dt, int N, int V, int64_t ldz, const int32_t* labels,
                           int32_t ignore_index, float* s, float* row_lse, int32_t* row_argmax, float* row_target,
                           void* R, int64_t ldr, float* loss, int32_t* n_valid, int32_t* flags, void* wsp,
                           hipStream_t stream) {
    const WsLayout L = ws_layout(N, V);
    char* base = static_cast<char*>(wsp);
    Partials ws{reinterpret_cast<float*>(base + L.part_off), reinterpret_cast<int*>(base + L.count_off),
                reinterpret_cast<int*>(base + L.flags_off), reinterpret_cast<double*>(base + L.loss_off),
                reinterpret_cast<unsigned long long*>(base + L.xch_off)};
    const int vw = dt == BOM_BF16 ? 8 : 4;
    const bool vec_ok = (ldz % vw == 0) && (reinterpret_cast<uintptr_t>(Z) % 16 == 0) &&
                        (R == nullptr || ((ldr % vw == 0) && reinterpret_cast<uintptr_t>(R) % 16 == 0)) &&
                        (V % vw == 0);
    if (dt == BOM_BF16) {
        const uint16_t* z = static_cast<const uint16_t*>(Z);
        uint16_t* r = static_cast<uint16_t*>(R);
        return vec_ok ? run_residual<uint16_t, 8>(z, N, V, ldz, labels, ignore_index, s, row_lse, row_argmax, row_target,
                                                  r, ldr, loss, n_valid, flags, ws, stream)
                      : run_residual<uint16_t, 1>(z, N, V, ldz, labels, ignore_index, s, row_lse, row_argmax, row_target,
                                                  r, ldr, loss, n_valid, flags, ws, stream);
    }
    const float* z = static_cast<const float*>(Z);
    float* r = static_cast<float*>(R);
    return vec_ok ? run_residual<float, 4>(z, N, V, ldz, labels, ignore_index, s, row_lse, row_argmax, row_target, r,
                                           ldr, loss, n_valid, flags, ws, stream)
                  : run_residual<float, 1>(z, N, V, ldz, labels, ignore_index, s, row_lse, row_argmax, row_target, r,
                                           ldr, loss, n_valid, flags, ws, stream);
}

// ---- allocation-free variant ----------------------------------------------------------------------
// A fixed device array that stands in for the caller's workspace (for callers that cannot allocate).
// Each device holds its own copy for the life of the process; host code never passes the array's name
// to a kernel (in host code it is a stand-in, not a device address): it looks up the device address once
// per device and passes that. Calls that overlap on one device share the array and race.
static __device__ __align__(256) unsigned char scratch[kResidualScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t residual_scratch(void** ptr) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr || reinterpret_cast<uintptr_t>(p) % 256 != 0) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return hipSuccess;
}

size_t residual_from_stats_workspace_bytes(int64_t N, int64_t V) { return stats_layout(N, V).total; }

// The row-statistics records live at the start of the workspace (written by launch_head_forward_stats).
hipError_t launch_residual_from_stats(const uint16_t* Z, int64_t ldz, int N, int V, const int32_t* labels,
                                      int32_t ignore_index, float* s, float* row_lse, int32_t* row_argmax,
                                      float* row_target, uint16_t* R, int64_t ldr, float* loss, int32_t* n_valid,
                                      int32_t* flags, void* wsp, hipStream_t st) {
    const StatsLayout L = stats_layout(N, V);
    char* base = static_cast<char*>(wsp);
    Partials ws{reinterpret_cast<float*>(base + L.part_off), reinterpret_cast<int*>(base + L.count_off),
                reinterpret_cast<int*>(base + L.flags_off), reinterpret_cast<double*>(base + L.loss_off), nullptr};
    hipLaunchKernelGGL(residual_combine_kernel, dim3((unsigned)L.nwg), dim3(kStatsRowsPerWG * kWave), 0, st,
                       reinterpret_cast<const float*>(base + L.stats_off), L.nT, N, V, labels, ignore_index, row_lse,
                       row_argmax, row_target, ws);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int slab = kColsThreads * kColsCPT * 8;
    dim3 grid((unsigned)(((V + slab - 1) / slab) * L.nparts));
    hipLaunchKernelGGL((residual_cols_kernel<uint16_t, 8>), grid, dim3(kColsThreads), 0, st, Z, ldz, N, V, labels,
                       ignore_index, row_lse, R, ldr, L.rb, ws.part);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(residual_finish_kernel, dim3((V + kWave - 1) / kWave), dim3(kFinThreads), 0, st, L.nparts, V, L.nwg,
                       ws, s, loss, n_valid, flags);
    return hipGetLastError();
}

}  // namespace bom
