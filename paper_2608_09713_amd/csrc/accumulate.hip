// Sparse sum of two lower parts, row by row: C = P + T with the union of the
// two patterns and the values of shared entries added (the stage accumulation
// C_ii = sum over stages of SYRK(A_is) of Sec. III-A, one stage at a time).
//
// Every row is a merge of two ascending column lists.  One pass counts each
// row's union, a scan gives the row pointers, a second pass writes the merged
// columns and sums.  A wavefront takes a row: each lane merges a contiguous
// part of the output found by a merge-path split (the lane's first output
// position is located in both lists by a binary search on the diagonal), so
// long rows spread over the lanes and short rows cost one pass.
#include "common.h"
#include "internal.h"

namespace spsyrk {
namespace {

constexpr int kRowsPerBlock = kWavesPerBlock;  // one row per wavefront
constexpr int kLdsRow = 512;                    // column ids of a list held in LDS

__device__ inline void wave_sync_acc() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int SR>
struct AccVal {
    using T = double;
};
template <>
struct AccVal<kF32> {
    using T = float;
};
template <>
struct AccVal<kCount> {
    using T = int32_t;
};

// Merge-path split of two ascending lists at position d of their merge with
// duplicates kept (a column in both lists appears twice, a's copy first):
// the number of a's entries among the merge's first d.
__device__ inline int64_t path_split(const int32_t* a, int64_t na, const int32_t* b, int64_t nb, int64_t d) {
    int64_t lo = d > nb ? d - nb : 0, hi = d < na ? d : na;
    while (lo < hi) {
        const int64_t ia = (lo + hi) >> 1;
        if (a[ia] <= b[d - 1 - ia])  // a[ia] precedes b[d - 1 - ia]: it is among the first d
            lo = ia + 1;
        else
            hi = ia;
    }
    return lo;
}

// Pass 1 (WRITE false): cnt[i] = distinct columns of row i of P and T.
// Pass 2 (WRITE true): the merged row at crp[i].  In the merge with
// duplicates kept, a column of both lists is a's copy followed by b's; b's
// copy is recognised by the a entry before it and writes nothing, and a's
// copy adds b's value (the next b entry when a's copy is taken).
template <int SR, bool WRITE>
__global__ __launch_bounds__(kBlock) void merge_rows(int64_t m, const int64_t* __restrict__ prp,
                                                     const int32_t* __restrict__ pci, const void* __restrict__ pv,
                                                     const int64_t* __restrict__ trp, const int32_t* __restrict__ tci,
                                                     const void* __restrict__ tv, int64_t* __restrict__ cnt,
                                                     const int64_t* __restrict__ crp, int32_t* __restrict__ cci,
                                                     void* __restrict__ cv) {
    using V = typename AccVal<SR>::T;
    __shared__ int32_t la[kRowsPerBlock][kLdsRow];
    __shared__ int32_t lb[kRowsPerBlock][kLdsRow];
    const int lane = lane_id();
    const int wv = threadIdx.x / kWave;
    const int64_t i = int64_t(blockIdx.x) * kRowsPerBlock + wv;
    if (i >= m) return;  // (whole wavefronts)
    const int64_t pa = prp[i], na = prp[i + 1] - pa;
    const int64_t ta = trp[i], nb = trp[i + 1] - ta;
    const int32_t* a = pci + pa;
    const int32_t* b = tci + ta;
    if (na <= kLdsRow && nb <= kLdsRow) {
        // short lists: staged in LDS by coalesced loads; the searches and the
        // merge below then read LDS
        for (int64_t t = lane; t < na; t += kWave) la[wv][t] = a[t];
        for (int64_t t = lane; t < nb; t += kWave) lb[wv][t] = b[t];
        wave_sync_acc();
        a = la[wv];
        b = lb[wv];
    }
    // the merge with duplicates kept, in equal parts over the lanes
    const int64_t total = na + nb;
    const int64_t per = (total + kWave - 1) / kWave;
    const int64_t d0 = min(total, per * lane), d1 = min(total, d0 + per);
    const int64_t ia0 = path_split(a, na, b, nb, d0), ib0 = d0 - ia0;
    const int64_t ia1 = path_split(a, na, b, nb, d1), ib1 = d1 - ia1;
    int64_t mine = 0;
    for (int64_t x = ia0, y = ib0; x < ia1 || y < ib1;) {
        if (y >= ib1 || (x < ia1 && a[x] <= b[y])) {
            ++mine;
            ++x;
        } else {
            if (!(x > 0 && a[x - 1] == b[y])) ++mine;
            ++y;
        }
    }
    const int64_t inc = wave_inclusive_scan(mine);
    if constexpr (!WRITE) {
        if (lane == kWave - 1) cnt[i] = inc;
    } else {
        int64_t out = crp[i] + inc - mine;
        const V* va = static_cast<const V*>(pv) + pa;
        const V* vb = static_cast<const V*>(tv) + ta;
        V* vc = static_cast<V*>(cv);
        for (int64_t x = ia0, y = ib0; x < ia1 || y < ib1;) {
            if (y >= ib1 || (x < ia1 && a[x] <= b[y])) {
                V v = va[x];
                if (y < nb && b[y] == a[x]) v = V(v + vb[y]);
                cci[out] = a[x];
                vc[out] = v;
                ++out;
                ++x;
            } else {
                if (!(x > 0 && a[x - 1] == b[y])) {
                    cci[out] = b[y];
                    vc[out] = vb[y];
                    ++out;
                }
                ++y;
            }
        }
    }
}

template <int SR>
void launch_merge(bool write, int64_t m, const DevCsr& P, const DevCsr& T, int64_t* cnt, const int64_t* crp,
                  int32_t* cci, void* cv, hipStream_t s) {
    const unsigned nb = unsigned((m + kRowsPerBlock - 1) / kRowsPerBlock);
    if (write)
        merge_rows<SR, true><<<nb, kBlock, 0, s>>>(m, P.rp, P.ci, P.v, T.rp, T.ci, T.v, cnt, crp, cci, cv);
    else
        merge_rows<SR, false><<<nb, kBlock, 0, s>>>(m, P.rp, P.ci, P.v, T.rp, T.ci, T.v, cnt, crp, cci, cv);
}

}  // namespace

void merge_lower(bool write, int sr, int64_t m, const DevCsr& P, const DevCsr& T, int64_t* cnt, const int64_t* crp,
                 int32_t* cci, void* cv, hipStream_t s) {
    if (m <= 0) return;
    switch (sr) {
        case kF64: launch_merge<kF64>(write, m, P, T, cnt, crp, cci, cv, s); break;
        case kF32: launch_merge<kF32>(write, m, P, T, cnt, crp, cci, cv, s); break;
        default: launch_merge<kCount>(write, m, P, T, cnt, crp, cci, cv, s); break;
    }
}

}  // namespace spsyrk
