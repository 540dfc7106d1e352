// Sparse sum of two lower parts, row by row: C = P + T with the union of the
// two patterns and the values of shared entries added (the stage accumulation
// C_ii = sum over stages of SYRK(A_is) of Sec. III-A, one stage at a time).
//
// The work is cut into items of at most kChunk entries of P and T together:
// chunks of consecutive short rows, and windows of kChunk merge positions of
// a long row.  A planning pass counts each row's items and a scan numbers
// them.  A workgroup takes an item.  It stages the item's entries in LDS as
// (row in the chunk, column) keys, so that its part of P and its part of T
// are two ascending lists, and merges them in equal parts over its threads: a
// thread's first output is located in both lists by a binary search on the
// merge diagonal (merge path); a window's own bounds are found the same way
// in the row's lists in global memory.  One pass counts each row's union, a
// scan gives the row pointers, a second pass writes the merged columns and
// sums.
#include "common.h"
#include "internal.h"

namespace spsyrk {
namespace {

constexpr int kLong = 256;                  // a row with more entries (P and T together) is split in windows
constexpr int kCapStart = 768;              // a chunk starts where (offset in P + offset in T) / kCapStart changes
constexpr int kChunk = kCapStart + kLong;   // entries of an item, at most (1024: about 20 KB of LDS,
                                            // so that eight workgroups share a compute unit)
constexpr int kRowCap = 1024;               // rows of a chunk, at most
static_assert(kRowCap <= kChunk, "the row marks' array holds the per-row counts");

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
// duplicates kept (a key in both lists appears twice, a's copy first): the
// number of a's entries among the merge's first d.
template <typename K, typename I>
__device__ inline I path_split(const K* a, I na, const K* b, I nb, I d) {
    I lo = d > nb ? d - nb : 0, hi = d < na ? d : na;
    while (lo < hi) {
        const I ia = (lo + hi) >> 1;
        if (a[ia] <= b[d - 1 - ia])  // a[ia] precedes b[d - 1 - ia]: it is among the first d
            lo = ia + 1;
        else
            hi = ia;
    }
    return lo;
}

// Walks the merge with duplicates kept from (x, y) to (x1, y1) and calls
// out(x, y) once per entry of the union: for a's entry x (y is then b's next
// entry, which holds the same key when b shares it), or with x = -1 for b's
// entry y when a does not hold its key.  A key of both lists is a's copy
// followed by b's; b's copy is recognised by the a entry before it.  a[-1]
// and b[nb] must be readable: the keys just outside the lists, or a key equal
// to no entry.
template <typename K, typename I, typename F>
__device__ inline void walk_union(const K* a, const K* b, I x, I y, I x1, I y1, F&& out) {
    while (x < x1 || y < y1) {
        if (y >= y1 || (x < x1 && a[x] <= b[y])) {
            out(x, y);
            ++x;
        } else {
            if (a[x - 1] != b[y]) out(I(-1), y);
            ++y;
        }
    }
}

// Work items of the merge.  Row i starts a chunk of short rows when it is the
// first row, a multiple of kRowCap, or the row after a long one, or when its
// offset s(i) (P's and T's offsets added) is in another kCapStart stretch than
// the previous row's; a chunk of short rows then holds fewer than kCapStart +
// kLong entries.  A long row (more than kLong entries) takes
// ceil(entries / kChunk) items, one per window of kChunk merge positions.
__device__ inline int64_t row_span(const int64_t* prp, const int64_t* trp, int64_t i) {
    return prp[i] - prp[0] + trp[i] - trp[0];
}

// fl[i] = items starting at row i; fl[m] = 0
__global__ __launch_bounds__(kBlock) void chunk_flags(int64_t m, const int64_t* __restrict__ prp,
                                                      const int64_t* __restrict__ trp, int64_t* __restrict__ fl) {
    const int64_t i = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (i > m) return;
    if (i == m) {
        fl[m] = 0;
        return;
    }
    const int64_t si = row_span(prp, trp, i), len = row_span(prp, trp, i + 1) - si;
    if (len > kLong) {
        fl[i] = (len + kChunk - 1) / kChunk;
        return;
    }
    bool f = i == 0 || i % kRowCap == 0;
    if (!f) {
        const int64_t sp = row_span(prp, trp, i - 1);
        f = si / kCapStart != sp / kCapStart || si - sp > kLong;
    }
    fl[i] = f ? 1 : 0;
}

// ex: exclusive scan of the flags (m + 1 words).  Item q: crow[q] = its first
// row, cwin[q] = its window of a long row, or -1 for a chunk of short rows
// (rows crow[q] to crow[q + 1]); crow[items] = m.
__global__ __launch_bounds__(kBlock) void chunk_items(int64_t m, const int64_t* __restrict__ prp,
                                                      const int64_t* __restrict__ trp,
                                                      const int64_t* __restrict__ ex, int64_t* __restrict__ crow,
                                                      int32_t* __restrict__ cwin) {
    const int64_t i = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (i > m) return;
    if (i == m) {
        crow[ex[m]] = m;
        return;
    }
    const int64_t q = ex[i], nq = ex[i + 1] - q;
    if (nq == 0) return;
    const bool lng = row_span(prp, trp, i + 1) - row_span(prp, trp, i) > kLong;
    for (int64_t k = 0; k < nq; ++k) {
        crow[q + k] = i;
        cwin[q + k] = lng ? int32_t(k) : -1;
    }
}

constexpr uint64_t kNone = ~uint64_t(0);  // a sentinel key equal to no entry

// Pass 1 (WRITE false): cnt[i] = distinct columns of row i of P and T (cnt
// zeroed before: a long row adds up its windows' counts), wsum[q] = the count
// of item q if it is a window, else 0.  Pass 2 (WRITE true, wsum scanned): the
// merged rows at crp.  One workgroup per item.  Its entries are staged in LDS
// as keys (row in the chunk << 32 | column): a sentinel, P's part, T's part,
// a second sentinel.  For a window the sentinels are the keys just outside
// it: they decide whether its first T entry repeats the P entry before it and
// whether its last P entry adds the T entry after it.
template <int SR, bool WRITE>
__global__ __launch_bounds__(kBlock) void merge_items(const int64_t* __restrict__ crow,
                                                      const int32_t* __restrict__ cwin,
                                                      const int64_t* __restrict__ prp,
                                                      const int32_t* __restrict__ pci, const void* __restrict__ pv,
                                                      const int64_t* __restrict__ trp,
                                                      const int32_t* __restrict__ tci, const void* __restrict__ tv,
                                                      int64_t* __restrict__ cnt, int64_t* __restrict__ wsum,
                                                      const int64_t* __restrict__ crp, int32_t* __restrict__ cci,
                                                      void* __restrict__ cv) {
    using V = typename AccVal<SR>::T;
    __shared__ uint64_t key[kChunk + 2];
    __shared__ V val[WRITE ? kChunk + 2 : 1];
    __shared__ uint32_t mark[kChunk];  // row marks, then the per-row counts
    __shared__ int64_t span[2];
    __shared__ uint32_t wt[kWavesPerBlock];
    const int tid = threadIdx.x;
    const int64_t item = blockIdx.x;
    const int64_t c0 = crow[item];
    const int win = cwin[item];
    const V* pvv = static_cast<const V*>(pv);
    const V* tvv = static_cast<const V*>(tv);
    int64_t pa, ta, na, nb, c1 = c0 + 1;
    uint64_t sa = kNone, sb = kNone;  // the sentinels
    V vsb = V(0);
    if (win < 0) {
        c1 = crow[item + 1];
        pa = prp[c0];
        ta = trp[c0];
        na = prp[c1] - pa;
        nb = trp[c1] - ta;
    } else {
        // merge positions [win * kChunk, +kChunk) of row c0, bounded by two
        // searches on the diagonals (the branch is uniform over the workgroup)
        const int64_t p0 = prp[c0], t0 = trp[c0], lp = prp[c0 + 1] - p0, lt = trp[c0 + 1] - t0;
        const int64_t d0 = int64_t(win) * kChunk, d1 = min(lp + lt, d0 + kChunk);
        if (tid == 0) span[0] = path_split(pci + p0, lp, tci + t0, lt, d0);
        if (tid == kWave) span[1] = path_split(pci + p0, lp, tci + t0, lt, d1);
        __syncthreads();
        const int64_t ia0 = span[0], ia1 = span[1], ib0 = d0 - ia0, ib1 = d1 - ia1;
        pa = p0 + ia0;
        ta = t0 + ib0;
        na = ia1 - ia0;
        nb = ib1 - ib0;
        if (ia0 > 0) sa = uint32_t(pci[pa - 1]);
        if (ib1 < lt) {
            sb = uint32_t(tci[ta + nb]);
            vsb = tvv[ta + nb];
        }
    }
    const int nA = int(na), nB = int(nb), n = nA + nB;
    const int nr = int(c1 - c0);
    for (int t = tid; t < n; t += kBlock) {
        key[1 + t] = uint32_t(t < nA ? pci[pa + t] : tci[ta + (t - nA)]);
        if constexpr (WRITE) val[1 + t] = t < nA ? pvv[pa + t] : tvv[ta + (t - nA)];
        if (win < 0) mark[t] = 0;
    }
    if (tid == 0) {
        key[0] = sa;
        key[1 + n] = sb;
        if constexpr (WRITE) val[1 + n] = vsb;
    }
    __syncthreads();
    if (win < 0) {
        // every non-empty part of a row marks its first entry; T's marks are
        // offset by kRowCap so that the max-scan below restarts at T's first
        // entry
        for (int r = tid; r < nr; r += kBlock) {
            const int64_t p0 = prp[c0 + r] - pa, p1 = prp[c0 + r + 1] - pa;
            if (p1 > p0) mark[p0] = uint32_t(r);
            const int64_t t0 = trp[c0 + r] - ta, t1 = trp[c0 + r + 1] - ta;
            if (t1 > t0) mark[nA + t0] = uint32_t(r + kRowCap);
        }
        __syncthreads();
        // a max-scan of the marks gives every entry's row
        const int per = (n + kBlock - 1) / kBlock;
        const int lo = min(n, tid * per), hi = min(n, lo + per);
        uint32_t mx = 0;
        for (int t = lo; t < hi; ++t) mx = max(mx, mark[t]);
        uint32_t all;
        uint32_t run = block_exclusive_max(mx, wt, &all);
        for (int t = lo; t < hi; ++t) {
            run = max(run, mark[t]);
            const uint32_t r = t < nA ? run : run - kRowCap;
            key[1 + t] |= uint64_t(r) << 32;
        }
        __syncthreads();
    }
    const uint64_t* a = key + 1;
    const uint64_t* b = key + 1 + nA;
    const int per = (n + kBlock - 1) / kBlock;
    const int d0 = min(n, tid * per), d1 = min(n, d0 + per);
    const int ia0 = path_split(a, nA, b, nB, d0), ib0 = d0 - ia0;
    const int ia1 = path_split(a, nA, b, nB, d1), ib1 = d1 - ia1;
    if constexpr (!WRITE) {
        if (win >= 0) {
            uint32_t mine = 0;
            walk_union(a, b, ia0, ib0, ia1, ib1, [&](int, int) { ++mine; });
            uint32_t tot;
            (void)block_exclusive_scan(mine, wt, &tot);
            if (tid == 0) {
                atomicAdd(reinterpret_cast<unsigned long long*>(cnt + c0), (unsigned long long)tot);
                wsum[item] = tot;
            }
            return;
        }
        if (tid == 0) wsum[item] = 0;
        uint32_t* rc = mark;
        for (int r = tid; r < nr; r += kBlock) rc[r] = 0;
        __syncthreads();
        uint32_t cur = 0, c = 0;
        walk_union(a, b, ia0, ib0, ia1, ib1, [&](int x, int y) {
            const uint32_t r = uint32_t((x >= 0 ? a[x] : b[y]) >> 32);
            if (r != cur) {
                if (c) atomicAdd(&rc[cur], c);
                cur = r;
                c = 0;
            }
            ++c;
        });
        if (c) atomicAdd(&rc[cur], c);
        __syncthreads();
        for (int r = tid; r < nr; r += kBlock) cnt[c0 + r] = rc[r];
    } else {
        uint32_t mine = 0;
        walk_union(a, b, ia0, ib0, ia1, ib1, [&](int, int) { ++mine; });
        uint32_t tot;
        int64_t o = crp[c0] + block_exclusive_scan(mine, wt, &tot);
        if (win >= 0) o += wsum[item] - wsum[item - win];  // the row's earlier windows
        V* vc = static_cast<V*>(cv);
        walk_union(a, b, ia0, ib0, ia1, ib1, [&](int x, int y) {
            if (x >= 0) {
                V v = val[1 + x];
                if (b[y] == a[x]) v = V(v + val[1 + nA + y]);
                cci[o] = int32_t(uint32_t(a[x]));
                vc[o] = v;
            } else {
                cci[o] = int32_t(uint32_t(b[y]));
                vc[o] = val[1 + nA + y];
            }
            ++o;
        });
    }
}

template <int SR>
void launch_merge(bool write, int64_t items, const int64_t* crow, const int32_t* cwin, const DevCsr& P,
                  const DevCsr& T, int64_t* cnt, int64_t* wsum, const int64_t* crp, int32_t* cci, void* cv,
                  hipStream_t s) {
    const unsigned nb = unsigned(items);
    if (write)
        merge_items<SR, true><<<nb, kBlock, 0, s>>>(crow, cwin, P.rp, P.ci, P.v, T.rp, T.ci, T.v, cnt, wsum, crp, cci,
                                                    cv);
    else
        merge_items<SR, false><<<nb, kBlock, 0, s>>>(crow, cwin, P.rp, P.ci, P.v, T.rp, T.ci, T.v, cnt, wsum, crp,
                                                     cci, cv);
}

}  // namespace

void merge_item_flags(int64_t m, const DevCsr& P, const DevCsr& T, int64_t* fl, void* scan_tmp, hipStream_t s) {
    if (m <= 0) return;
    const unsigned g = unsigned((m + 1 + kBlock - 1) / kBlock);
    chunk_flags<<<g, kBlock, 0, s>>>(m, P.rp, T.rp, fl);
    scan_i64(fl, fl, m + 1, nullptr, scan_tmp, s);
}

void merge_item_table(int64_t m, const DevCsr& P, const DevCsr& T, const int64_t* fl, int64_t* crow, int32_t* cwin,
                      hipStream_t s) {
    if (m <= 0) return;
    const unsigned g = unsigned((m + 1 + kBlock - 1) / kBlock);
    chunk_items<<<g, kBlock, 0, s>>>(m, P.rp, T.rp, fl, crow, cwin);
}

void merge_lower(bool write, int sr, int64_t items, const int64_t* crow, const int32_t* cwin, const DevCsr& P,
                 const DevCsr& T, int64_t* cnt, int64_t* wsum, const int64_t* crp, int32_t* cci, void* cv,
                 hipStream_t s) {
    if (items <= 0) return;
    switch (sr) {
        case kF64: launch_merge<kF64>(write, items, crow, cwin, P, T, cnt, wsum, crp, cci, cv, s); break;
        case kF32: launch_merge<kF32>(write, items, crow, cwin, P, T, cnt, wsum, crp, cci, cv, s); break;
        default: launch_merge<kCount>(write, items, crow, cwin, P, T, cnt, wsum, crp, cci, cv, s); break;
    }
}

}  // namespace spsyrk
