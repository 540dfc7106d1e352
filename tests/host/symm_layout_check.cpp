// Host check of the bucket layout of the product from a stored lower part:
// for every row count up to 2^24 around powers of two and every setting of
// the bucket choice, a bucketed product never has more buckets than the LDS
// tables hold, and the bucket size stays in 2^12 .. 2^14 rows.
#include <cstdio>
#include <cstdint>
#include <initializer_list>

#include "symm_layout.h"

int main() {
    using namespace spsyrk;
    long checked = 0, bucketed = 0;
    const int settings[] = {-1, 0, 1, 12, 13, 14};
    for (int p = 0; p <= 25; ++p) {
        for (int64_t d = -3; d <= 3; ++d) {
            const int64_t m = (int64_t(1) << p) + d;
            if (m < 1) continue;
            for (int f : settings) {
                ++checked;
                if (!symm_bucketed(m, 1, 10, f)) {
                    if (f == 1 && m <= kSymmMaxBucketRows) {
                        std::printf("forced buckets refused at m=%lld\n", (long long)m);
                        return 1;
                    }
                    continue;
                }
                ++bucketed;
                const int bits = symm_bucket_bits(m, f);
                const int nbk = symm_bucket_count(m, bits);
                if (bits < 12 || bits > 14 || nbk > kSymmMaxBuckets || nbk < 1 ||
                    (int64_t(nbk) << bits) < m) {
                    std::printf("bad layout m=%lld forced=%d bits=%d buckets=%d\n", (long long)m, f, bits, nbk);
                    return 1;
                }
                if (f >= 12 && m <= (int64_t(1024) << f) && bits != f) {
                    std::printf("forced %d changed to %d at m=%lld\n", f, bits, (long long)m);
                    return 1;
                }
            }
            // more than one column never takes buckets
            if (symm_bucketed(m, 2, 10, 1)) return 1;
        }
    }
    // the range split: ranges of at most 2^14 rows (the LDS accumulator), at
    // most kSymmSplitMax of them, covering all m rows
    for (int p = 0; p <= 31; ++p) {
        for (int64_t d = -1; d <= 1; ++d) {
            const int64_t m = (int64_t(1) << p) + d;
            if (m < 1) continue;
            for (int f : {0, 1, 8, 10, 14, 20}) {
                const int bits = symm_split_bits(m, f);
                const int64_t nr = (m + (int64_t(1) << bits) - 1) >> bits;
                const bool on = symm_split(m, 1, 10, 1, f);
                if (bits < 1 || bits > kSymmSplitBits || (on && (nr < 1 || nr > kSymmSplitMax))) {
                    std::printf("bad split m=%lld forced=%d bits=%d ranges=%lld\n", (long long)m, f, bits, (long long)nr);
                    return 1;
                }
                if (symm_split(m, 2, 10, 1, f)) return 1;  // one column only
            }
        }
    }
    std::printf("ok %ld settings, %ld bucketed\n", checked, bucketed);
    return 0;
}
