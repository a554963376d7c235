// na_fastdiv.h -- division by a divisor fixed for a whole launch or
// workgroup, as a multiply and a shift (Granlund and Montgomery, "Division by
// Invariant Integers using Multiplication", PLDI 1994: the round-up method
// with a 33-bit multiplier 2^32 + mul, whose top bit becomes the "+ n").
//
// For 1 <= d < 2^31 and 0 <= n < 2^31:
//   s   = ceil(log2 d)
//   mul = floor(2^32 (2^s - d) / d) + 1
//   n / d = (umulhi(n, mul) + n) >> s
// (umulhi(n, mul) < 2^31, so the sum stays below 2^32.)  The multiplier is
// formed on the host in 64-bit integers; on the device it is 1 for a power of
// two (2^s - d = 0) and otherwise, for d < 2^20, comes from one double
// division (2^32 (2^s - d) < 2^52 is exact in a double,
// the division is correctly rounded, and the quotient's fractional part is at
// least 1/d > 2^-20, far above the rounding error of a quotient below 2^32, so
// its floor is exact).  Both paths are plain C++ here so that a host build
// can check them against each other and against integer division.
#pragma once

#include <stdint.h>

#include "na_index.h"

namespace na {

struct FastDiv {
    uint32_t mul, shr;

    static NA_HD uint32_t shift_for(int d) {  // ceil(log2 d)
        return d <= 1 ? 0u : 32u - (uint32_t)__builtin_clz((uint32_t)d - 1u);
    }
    // multiplier from 64-bit integers (any 1 <= d < 2^31)
    static NA_HD uint32_t mul_int(int d, uint32_t s) {
        const uint64_t a = ((uint64_t)1 << s) - (uint64_t)d;
        return (uint32_t)((a << 32) / (uint64_t)d + 1);
    }
    // multiplier from one double division (1 <= d < 2^20)
    static NA_HD uint32_t mul_double(int d, uint32_t s) {
        const uint64_t a = ((uint64_t)1 << s) - (uint64_t)d;
        return (uint32_t)((uint64_t)__builtin_floor((double)a * 4294967296.0 / (double)d) + 1);
    }

    NA_HD void init(int d) {
        shr = shift_for(d);
#if defined(__HIP_DEVICE_COMPILE__)
        // a power of two (2^s - d = 0): the multiplier is 1, so no division at
        // all -- the common case of the per-workgroup divisors
        if ((d & (d - 1)) == 0) {
            mul = 1;
            return;
        }
        if (d < (1 << 20)) {
            mul = mul_double(d, shr);
            return;
        }
#endif
        mul = mul_int(d, shr);
    }

    static NA_HD int divide(int n, uint32_t mul, uint32_t shr) {
#if defined(__HIP_DEVICE_COMPILE__)
        return (int)((__umulhi((uint32_t)n, mul) + (uint32_t)n) >> shr);
#else
        const uint32_t hi = (uint32_t)(((uint64_t)(uint32_t)n * mul) >> 32);
        return (int)((hi + (uint32_t)n) >> shr);
#endif
    }
    NA_HD int div(int n) const { return divide(n, mul, shr); }
};

}  // namespace na
