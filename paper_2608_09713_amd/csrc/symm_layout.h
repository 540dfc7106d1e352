// Host-side choice of the paths of the product from a stored lower part with
// one column: whether the transposed term goes through LDS buckets of rows
// (and how many rows a bucket holds) or through records split by row range.  Plain C++ (no HIP), so that the
// choice can be checked on any host.
#pragma once

#include <cstdint>

namespace spsyrk {

// at most this many buckets: the counting and record passes keep one LDS
// counter or cursor per bucket
constexpr int kSymmMaxBuckets = 1024;
// bucketed products have at most this many rows
constexpr int64_t kSymmMaxBucketRows = int64_t(1) << 24;

// ceil(log2 m) for m >= 1
inline int symm_ceil_log2(int64_t m) {
    int b = 0;
    while ((int64_t(1) << b) < m) ++b;
    return b;
}

// log2 of the rows per bucket, from 12 to 14.  Unforced: about 256 buckets
// (ceil(log2 m) - 8).  Forced (12, 13 or 14): that value, raised where needed
// so that the buckets never number more than kSymmMaxBuckets.
inline int symm_bucket_bits(int64_t m, int forced) {
    const int lg = symm_ceil_log2(m < 1 ? 1 : m);
    int bits = forced >= 12 ? forced : lg - 8;
    if (bits < lg - 10) bits = lg - 10;  // ceil(m / 2^bits) <= 1024
    return bits < 12 ? 12 : (bits > 14 ? 14 : bits);
}

inline int symm_bucket_count(int64_t m, int bits) { return int((m + (int64_t(1) << bits) - 1) >> bits); }

// forced: -1 unforced, 0 never, 1 always (up to kSymmMaxBucketRows rows),
// 12..14 always with that bucket size.  Unforced, buckets serve a single
// column of 2^19 to 2^21 rows.
inline bool symm_bucketed(int64_t m, int64_t k, int64_t nnz, int forced) {
    if (k != 1 || nnz <= 0 || m > kSymmMaxBucketRows || forced == 0) return false;
    if (forced < 0 && !(m > (int64_t(1) << 19) && m <= (int64_t(1) << 21))) return false;
    return symm_bucket_count(m, symm_bucket_bits(m, forced)) <= kSymmMaxBuckets;
}

// Split path of a single column past 2^21 rows: the transposed terms are
// written as records grouped by ranges of 2^bits rows of Y (2^14 rows, a
// 128 KiB accumulator of doubles in LDS; at most kSymmSplitMax ranges), each
// tile's records sorted by range so that every range gets one contiguous run,
// then every range summed in LDS.
constexpr int kSymmSplitMax = 1024;
constexpr int kSymmSplitBits = 14;

// forced: 0 for the default 2^14 rows per range, else that many bits (at
// most 14)
inline int symm_split_bits(int64_t, int forced) {
    return forced > 0 && forced < kSymmSplitBits ? forced : kSymmSplitBits;
}

// forced: -1 unforced (past 2^21 rows), 0 never, 1 always (single columns);
// never past kSymmSplitMax ranges of the range size
inline bool symm_split(int64_t m, int64_t k, int64_t nnz, int forced, int forced_bits = 0) {
    if (k != 1 || nnz <= 0 || m <= 0 || forced == 0) return false;
    const int bits = symm_split_bits(m, forced_bits);
    if (((m + (int64_t(1) << bits) - 1) >> bits) > kSymmSplitMax) return false;
    return forced == 1 || m > (int64_t(1) << 21);
}

}  // namespace spsyrk
