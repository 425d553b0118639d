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

// The 56 masks made of the centre and 3 of its 8 neighbours, ascending: the
// shapes the pattern heuristic of Sec. 4.2 can produce, for which the conv
// kernels have loops compiled with their taps fixed.
struct Centre3Table {
    uint16_t code[56];
    constexpr Centre3Table() : code{} {
        int n = 0;
        for (int c = 0; c < 512; ++c) {
            int pc = 0;
            for (int b = 0; b < 9; ++b) pc += (c >> b) & 1;
            if (((c >> 4) & 1) && pc == 4) code[n++] = uint16_t(c);
        }
    }
};
constexpr Centre3Table kCentre3{};

// Position of the JJ-th set bit of MASK (ascending), -1 if none.
template <int MASK, int JJ>
struct NthBit {
    static constexpr int value() {
        int seen = 0;
        for (int q = 0; q < 9; ++q)
            if ((MASK >> q) & 1) {
                if (seen == JJ) return q;
                ++seen;
            }
        return -1;
    }
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
