// Small device-side helpers shared by the copy kernels of the library.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>

#include "plan.hpp"

namespace remp {

// Division by a runtime constant d for any 32-bit numerator (Granlund and
// Montgomery, "Division by invariant integers using multiplication", 1994):
// with l = ceil(log2 d) and m = floor(2^32 (2^l - d) / d) + 1,
// n / d = (mulhi(m, n) + n) >> l, the sum taken in 33 bits.
struct FastDiv {
    uint32_t magic;
    uint32_t shift;
};

inline FastDiv make_fastdiv(uint32_t d) {
    uint32_t l = 0;
    while ((uint64_t(1) << l) < d) ++l;
    uint64_t m = ((uint64_t(1) << 32) * ((uint64_t(1) << l) - d)) / d + 1;
    return FastDiv{static_cast<uint32_t>(m), l};
}

__device__ __forceinline__ uint32_t fast_div(uint32_t n, uint32_t magic, uint32_t shift) {
    uint64_t t = __umulhi(n, magic);
    return static_cast<uint32_t>((t + n) >> shift);
}

// Vector type of VEC bytes moved by one load / store.
template <int VEC> struct VecT;
template <> struct VecT<16> { typedef unsigned int type __attribute__((ext_vector_type(4))); };
template <> struct VecT<8> { typedef unsigned int type __attribute__((ext_vector_type(2))); };
template <> struct VecT<4> { typedef unsigned int type; };
template <> struct VecT<2> { typedef unsigned short type; };
template <> struct VecT<1> { typedef unsigned char type; };

inline remp_status hip_check(hipError_t e, const char* what) {
    if (e == hipSuccess) return REMP_OK;
    return fail(REMP_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

}  // namespace remp
