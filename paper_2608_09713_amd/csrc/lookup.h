// Partner-run lookup in the column index of the right operand.
#pragma once

#include "common.h"
#include "internal.h"

namespace spsyrk {

// For the stored entry (i, k) of the left operand, the partners are the
// entries of column k of the right operand B: all of them off the diagonal,
// only those with row j < i for the lower triangle (Sec. III-A computes the
// lower triangle of a diagonal block).  Inside a column the keys ascend with
// the row, so the partners are one contiguous run [start, start + len).
__device__ inline void partner_run(const uint32_t* __restrict__ key, const uint32_t* __restrict__ gptr, int gs,
                                   int rowbits, uint32_t k, uint32_t i, bool lower, uint32_t& start, uint32_t& len) {
    const uint32_t g = gs >= 32 ? 0u : (k >> gs);
    const int64_t lo = gptr[g];
    const int64_t hi = gptr[g + 1];
    const uint32_t gmask = gs >= 32 ? 0xffffffffu : ((1u << gs) - 1u);
    const uint64_t klo = uint64_t(k & gmask) << rowbits;
    const int64_t p0 = lower_bound_u32(key, lo, hi, klo);
    const uint64_t kend = lower ? (klo | uint64_t(i)) : (klo + (uint64_t(1) << rowbits));
    const int64_t p1 = lower_bound_u32(key, p0, hi, kend);
    start = uint32_t(p0);
    len = uint32_t(p1 - p0);
}

template <int SR>
struct SrTraits;

// plus-times over double
template <>
struct SrTraits<kF64> {
    using In = double;      // value type of A and of the column index
    using Item = double;    // per-product payload
    using Acc = double;     // dense accumulator
    using Out = double;
    static constexpr bool kHasItem = true;
};
// plus-times over float inputs, double products and sums, float output
template <>
struct SrTraits<kF32> {
    using In = float;
    using Item = double;
    using Acc = double;
    using Out = float;
    static constexpr bool kHasItem = true;
};
// shared-column count
template <>
struct SrTraits<kCount> {
    using In = float;       // unused
    using Item = int32_t;   // unused
    using Acc = int32_t;
    using Out = int32_t;
    static constexpr bool kHasItem = false;
};
// shared-column count finalised to Jaccard; the item carries |S(j)|
template <>
struct SrTraits<kJaccard> {
    using In = float;       // unused
    using Item = int32_t;
    using Acc = int32_t;
    using Out = float;
    static constexpr bool kHasItem = true;
};

// J = c / (|a| + |b| - c), one correctly rounded float division.  Row
// lengths are below 2^31, so the denominator fits 32 unsigned bits, whose
// conversion rounds as the 64-bit one would.
__device__ inline float jaccard(int32_t c, int64_t len_a, int64_t len_b) {
    const uint32_t d = uint32_t(len_a) + uint32_t(len_b) - uint32_t(c);
    return __fdiv_rn(float(c), float(d));
}

}  // namespace spsyrk
