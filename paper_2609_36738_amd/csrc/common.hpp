// Device helpers shared by the BOM kernels (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bom.h"

namespace bom {

constexpr int kWave = 64;

// Native 4-wide vector (the non-temporal load/store builtins take clang vector types).
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Streaming (non-temporal) 16-byte accesses: data read or written once per launch.
__device__ __forceinline__ f32x4 ld_stream(const float* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
}
__device__ __forceinline__ void st_stream(float* p, f32x4 v) {
    __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(p));
}

// All-ones / zero lane mask, opaque to the optimiser. A load followed by `& lane_mask(ok)` stays an
// unconditional load: the compiler cannot sink it into a branch (which would serialise the loads of
// a tile behind a wait for each one).
__device__ __forceinline__ uint32_t lane_mask(bool ok) {
    uint32_t m = ok ? 0xFFFFFFFFu : 0u;
    asm("" : "+v"(m));  // not volatile: opaque, but free to schedule
    return m;
}
__device__ __forceinline__ uint4 and_mask(uint4 v, uint32_t m) { return make_uint4(v.x & m, v.y & m, v.z & m, v.w & m); }

// ---- bf16 <-> fp32 (bf16 is carried as raw uint16_t) ----------------------------------------
__device__ __forceinline__ float bf16_lo(uint32_t packed) { return __uint_as_float(packed << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t packed) { return __uint_as_float(packed & 0xFFFF0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t x) { return __uint_as_float((uint32_t)x << 16); }

// Round-to-nearest-even fp32 -> bf16 pair; gfx950 does this in one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
    bf16x2_t v;
    v[0] = (__bf16)lo;
    v[1] = (__bf16)hi;
    return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ uint16_t f32_to_bf16(float x) {
    __bf16 v = (__bf16)x;
    return __builtin_bit_cast(uint16_t, v);
}

// ---- wave reductions (xor butterflies over 64 lanes) -------------------------------------
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}
__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}
__device__ __forceinline__ int wave_min(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o, kWave));
    return v;
}
__device__ __forceinline__ int wave_or(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v |= __shfl_xor(v, o, kWave);
    return v;
}

// ---- reductions with DPP lane permutes (VALU only: no LDS round trip per step) -------------
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
// Every lane of each 16-lane row ends with the row's maximum (sum): partners at xor 1 and xor 2 (quad
// permutes 0xB1, 0x4E), then the other quad of each eight (half mirror, 0x141) and the other eight of
// the sixteen (mirror, 0x140). Each step combines two lanes that hold the same partial in either
// order, so all lanes of a row end with the same bits.
__device__ __forceinline__ float row16_max(float v) {
    v = fmaxf(v, dpp_f32<0xB1>(v));
    v = fmaxf(v, dpp_f32<0x4E>(v));
    v = fmaxf(v, dpp_f32<0x141>(v));
    return fmaxf(v, dpp_f32<0x140>(v));
}
__device__ __forceinline__ float row16_sum(float v) {
    v += dpp_f32<0xB1>(v);
    v += dpp_f32<0x4E>(v);
    v += dpp_f32<0x141>(v);
    return v + dpp_f32<0x140>(v);
}
__device__ __forceinline__ float lane_f32(float v, int lane) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}
// wave-uniform maximum and sum: the four row results combined as ((r0, r1), (r2, r3))
__device__ __forceinline__ float wave_max_dpp(float v) {
    v = row16_max(v);
    return fmaxf(fmaxf(lane_f32(v, 0), lane_f32(v, 16)), fmaxf(lane_f32(v, 32), lane_f32(v, 48)));
}
__device__ __forceinline__ float wave_sum_dpp(float v) {
    v = row16_sum(v);
    return (lane_f32(v, 0) + lane_f32(v, 16)) + (lane_f32(v, 32) + lane_f32(v, 48));
}
__device__ __forceinline__ int wave_min_dpp(int v) {
    v = min(v, __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false));
    v = min(v, __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false));
    v = min(v, __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false));
    v = min(v, __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false));
    return min(min(__builtin_amdgcn_readlane(v, 0), __builtin_amdgcn_readlane(v, 16)),
               min(__builtin_amdgcn_readlane(v, 32), __builtin_amdgcn_readlane(v, 48)));
}

// exp and log with the hardware base-2 units: exp(x) = 2^(x log2 e).
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ bool label_valid(int32_t y, int64_t V, int32_t ignore_index, bool* bad) {
    if (y == ignore_index) return false;
    if (y < 0 || (int64_t)y >= V) {
        *bad = true;
        return false;
    }
    return true;
}

constexpr int kBufFlags = 0x00020000;   // raw buffer descriptor word 3: 32-bit data format
constexpr int kOob = (int)0x80000000u;  // an offset past every range: the load returns zeros
constexpr int kNonTemporal = 2;           // buffer access cache policy: nt (streamed data touched once)

typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
typedef int i32x4_t __attribute__((ext_vector_type(4)));   // buffer descriptor words for inline assembly

// Raw buffer descriptor over [base, base + bytes): loads at offsets >= bytes return zeros and
// stores there are dropped.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_desc(const void* base, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, kBufFlags);
}

}  // namespace bom
