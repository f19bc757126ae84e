/*
 * Seeded synthetic-input generators shared by the tests, the benchmark and the
 * smoke check. This file holds no arithmetic of the optimizer: it only turns
 * (seed, stream, element index) into numbers.
 *
 * Generator: Philox4x32-10, the counter-based generator of Salmon, Moraes,
 * Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3" (SC'11).
 * Key = the 64-bit seed split into two 32-bit words; counter = (index low
 * word, index high word, stream id, 0). Because every value depends only on
 * its own counter, any slice of any tensor can be regenerated on its own.
 *
 * Normals: Box-Muller in fp64 on two 53-bit uniforms in (0, 1]; the pair
 * index e/2 selects the counter, even elements take the cosine branch and odd
 * elements the sine branch. The fp64 value times `std` is rounded to fp32
 * (round-to-nearest-even), and for bf16 tensors that fp32 value is rounded
 * again to bf16 (round-to-nearest-even).
 *
 * Labels: uniform over C classes as floor(x * C / 2^64) for a 64-bit draw x;
 * or truncated Zipf with P(rank k) proportional to k^-a for k = 1..V, sampled
 * by inverse CDF on an fp64 table, label = k - 1.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

static inline void philox4x32_10(const uint32_t in[4], const uint32_t key_in[2], uint32_t out[4]) {
    uint32_t x0 = in[0], x1 = in[1], x2 = in[2], x3 = in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int r = 0; r < 10; ++r) {
        uint64_t p0 = (uint64_t)PHILOX_M0 * x0;
        uint64_t p1 = (uint64_t)PHILOX_M1 * x2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t y0 = hi1 ^ x1 ^ k0;
        uint32_t y1 = lo1;
        uint32_t y2 = hi0 ^ x3 ^ k1;
        uint32_t y3 = lo0;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
        k0 += PHILOX_W0;
        k1 += PHILOX_W1;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

static inline void draw(uint64_t seed, uint32_t stream, uint64_t index, uint32_t out[4]) {
    uint32_t ctr[4] = {(uint32_t)index, (uint32_t)(index >> 32), stream, 0u};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    philox4x32_10(ctr, key, out);
}

/* 53-bit uniform in (0, 1]. */
static inline double u53(uint32_t hi, uint32_t lo) {
    uint64_t x = (((uint64_t)hi << 32) | lo) >> 11;
    return (double)(x + 1) * (1.0 / 9007199254740992.0);
}

static inline double normal_at(uint64_t seed, uint32_t stream, uint64_t e) {
    uint32_t o[4];
    draw(seed, stream, e >> 1, o);
    double u1 = u53(o[0], o[1]);
    double u2 = u53(o[2], o[3]);
    double rad = sqrt(-2.0 * log(u1));
    double ang = 6.283185307179586476925286766559 * u2;
    return (e & 1) ? rad * sin(ang) : rad * cos(ang);
}

static inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t b;
    memcpy(&b, &f, 4);
    if ((b & 0x7F800000u) == 0x7F800000u && (b & 0x007FFFFFu)) return (uint16_t)((b >> 16) | 0x40u);
    uint32_t lsb = (b >> 16) & 1u;
    b += 0x7FFFu + lsb;
    return (uint16_t)(b >> 16);
}

/* Known-answer access to the raw generator. */
void synth_philox(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0, uint32_t k1,
                  uint32_t* out4) {
    uint32_t ctr[4] = {c0, c1, c2, c3};
    uint32_t key[2] = {k0, k1};
    philox4x32_10(ctr, key, out4);
}

/* out[i] = fp32(std * normal(start + i)), i in [0, n). */
void synth_normal_f32(float* out, int64_t n, int64_t start, uint64_t seed, uint32_t stream, double std) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = (float)(std * normal_at(seed, stream, (uint64_t)(start + i)));
}

/* Same values as synth_normal_f32, rounded once more to bf16; returned as raw 16-bit patterns. */
void synth_normal_bf16(uint16_t* out, int64_t n, int64_t start, uint64_t seed, uint32_t stream, double std) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        float f = (float)(std * normal_at(seed, stream, (uint64_t)(start + i)));
        out[i] = f32_to_bf16_rne(f);
    }
}

/* Uniform labels in [0, C). */
void synth_labels_uniform(int32_t* out, int64_t n, int64_t start, uint64_t seed, uint32_t stream, int64_t C) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        uint32_t o[4];
        draw(seed, stream, (uint64_t)(start + i), o);
        uint64_t x = ((uint64_t)o[0] << 32) | o[1];
        out[i] = (int32_t)(((unsigned __int128)x * (unsigned __int128)(uint64_t)C) >> 64);
    }
}

/* Truncated Zipf(a) over V labels. */
int synth_labels_zipf(int32_t* out, int64_t n, int64_t start, uint64_t seed, uint32_t stream, int64_t V, double a) {
    double* cdf = (double*)malloc((size_t)V * sizeof(double));
    if (!cdf) return -1;
    double acc = 0.0;
    for (int64_t k = 0; k < V; ++k) {
        acc += pow((double)(k + 1), -a);
        cdf[k] = acc;
    }
    for (int64_t k = 0; k < V; ++k) cdf[k] /= acc;
    cdf[V - 1] = 1.0;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        uint32_t o[4];
        draw(seed, stream, (uint64_t)(start + i), o);
        double u = u53(o[0], o[1]);
        int64_t lo = 0, hi = V - 1;
        while (lo < hi) {
            int64_t mid = lo + (hi - lo) / 2;
            if (cdf[mid] >= u) hi = mid; else lo = mid + 1;
        }
        out[i] = (int32_t)lo;
    }
    free(cdf);
    return 0;
}

/* Uniform (0, 1] doubles, for masks such as the ignored-target variant. */
void synth_uniform_f64(double* out, int64_t n, int64_t start, uint64_t seed, uint32_t stream) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        uint32_t o[4];
        draw(seed, stream, (uint64_t)(start + i), o);
        out[i] = u53(o[0], o[1]);
    }
}

/* bf16 raw patterns -> fp32 (exact widening). */
void synth_bf16_to_f32(const uint16_t* in, float* out, int64_t n) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        uint32_t b = (uint32_t)in[i] << 16;
        memcpy(&out[i], &b, 4);
    }
}
