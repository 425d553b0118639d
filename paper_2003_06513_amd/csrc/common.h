// Shared device-side definitions for the psc kernels (product code only).
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

namespace psc {

enum : int { DT_F32 = 0, DT_F16 = 1 };
constexpr int kMaxPatterns = 126;

// The pattern library as a kernel argument (Sec. 3.2: m masks of 4 kept
// positions, bit 3r+s).
struct PatTable {
    int32_t m;
    uint16_t mask[kMaxPatterns];
};

// Storage <-> fp32 conversions.  fp16 is IEEE binary16; widening is exact,
// narrowing rounds to nearest even (the hardware default mode).
template <int DT> struct Elt;
template <> struct Elt<DT_F32> {
    using T = float;
    using Bits = uint32_t;
    __device__ __forceinline__ static float load(const T* p, int64_t i) { return p[i]; }
    __device__ __forceinline__ static T from_f(float v) { return v; }
};
template <> struct Elt<DT_F16> {
    using T = uint16_t;
    using Bits = uint16_t;
    __device__ __forceinline__ static float load(const T* p, int64_t i) {
        return (float)__builtin_bit_cast(_Float16, p[i]);
    }
    __device__ __forceinline__ static T from_f(float v) {
        return __builtin_bit_cast(uint16_t, (_Float16)v);
    }
};

}  // namespace psc
