// Vectorised row I/O for fp32 and bf16 (raw uint16_t) rows: 16-byte accesses when the row pitch
// and base allow it, scalar accesses otherwise (and for the ragged last chunk of a row).
#pragma once
#include "common.hpp"

namespace bom {

template <typename T, int VEC>
struct VecIO;

template <>
struct VecIO<uint16_t, 8> {
    static __device__ __forceinline__ void load(const uint16_t* p, float* x) {
        uint4 u = *reinterpret_cast<const uint4*>(p);
        x[0] = bf16_lo(u.x); x[1] = bf16_hi(u.x);
        x[2] = bf16_lo(u.y); x[3] = bf16_hi(u.y);
        x[4] = bf16_lo(u.z); x[5] = bf16_hi(u.z);
        x[6] = bf16_lo(u.w); x[7] = bf16_hi(u.w);
    }
    static __device__ __forceinline__ void store(uint16_t* p, const float* x) {
        uint4 u;
        u.x = pack_bf16x2(x[0], x[1]);
        u.y = pack_bf16x2(x[2], x[3]);
        u.z = pack_bf16x2(x[4], x[5]);
        u.w = pack_bf16x2(x[6], x[7]);
        *reinterpret_cast<uint4*>(p) = u;
    }
};

template <>
struct VecIO<float, 4> {
    static __device__ __forceinline__ void load(const float* p, float* x) {
        float4 u = *reinterpret_cast<const float4*>(p);
        x[0] = u.x; x[1] = u.y; x[2] = u.z; x[3] = u.w;
    }
    static __device__ __forceinline__ void store(float* p, const float* x) {
        *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
    }
};

template <>
struct VecIO<uint16_t, 1> {
    static __device__ __forceinline__ void load(const uint16_t* p, float* x) { x[0] = bf16_to_f32(*p); }
    static __device__ __forceinline__ void store(uint16_t* p, const float* x) { *p = f32_to_bf16(x[0]); }
};

template <>
struct VecIO<float, 1> {
    static __device__ __forceinline__ void load(const float* p, float* x) { x[0] = *p; }
    static __device__ __forceinline__ void store(float* p, const float* x) { *p = x[0]; }
};

template <typename T>
__device__ __forceinline__ float load_scalar(const T* p);
template <>
__device__ __forceinline__ float load_scalar<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float load_scalar<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }

template <typename T>
__device__ __forceinline__ void store_scalar(T* p, float x);
template <>
__device__ __forceinline__ void store_scalar<float>(float* p, float x) { *p = x; }
template <>
__device__ __forceinline__ void store_scalar<uint16_t>(uint16_t* p, float x) { *p = f32_to_bf16(x); }

// Load VEC consecutive elements starting at column `col` (a multiple of VEC) of a row whose
// length V is a multiple of VEC, so a chunk is wholly inside or wholly outside the row;
// outside chunks read as `fill`.
// The load itself is unconditional (a clamped in-range address), so the compiler keeps every chunk's
// load in flight together instead of sinking each one into a branch.
template <typename T, int VEC>
__device__ __forceinline__ void load_chunk(const T* row, int col, int V, float fill, float* x) {
    const bool ok = col < V;
    VecIO<T, VEC>::load(row + (ok ? col : V - VEC), x);
    const uint32_t m = lane_mask(ok);
    const uint32_t fb = __float_as_uint(fill) & ~m;
#pragma unroll
    for (int k = 0; k < VEC; ++k) x[k] = __uint_as_float((__float_as_uint(x[k]) & m) | fb);
}

template <typename T, int VEC>
__device__ __forceinline__ void store_chunk(T* row, int col, int V, const float* x) {
    if (col < V) VecIO<T, VEC>::store(row + col, x);
}

}  // namespace bom
