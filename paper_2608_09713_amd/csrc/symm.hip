// Y = C X for the symmetric C = C_L + C_L^T - D, read from the stored lower
// part only (Eq. (spmv), and Eq. (spgemm) for several columns): each stored
// C_L(i, j) adds C_L(i, j) X(j, :) to Y(i, :) (the product with C_L) and, off
// the diagonal, C_L(i, j) X(i, :) to Y(j, :) (the vector-times-matrix term
// X^T C_L, transposed); the diagonal counts once, which is the - D X.
//
// One pass over C_L in tiles of consecutive entries; every group of lanes
// walks a stretch of entries row by row (rows found in an LDS window of the
// row pointers, as the row-product kernel does), one lane per column of X.  The row term is summed per row
// stretch and added once; the transposed term is a scatter of atomic adds.
// Everything accumulates in double in a zeroed m x k workspace, which a last
// pass rounds into Y.
//
// For a single column (the product with a vector) the transposed term's
// random atomic adds miss in L2 and bound the whole pass, so they are
// bucketed instead: rows of Y are grouped in buckets of 2^12 to 2^14 rows; a counting
// pass sizes every (bucket, workgroup) stretch of a bucket-major record array,
// the row pass writes each term as a record (row in the bucket, value) into
// its stretch, and a last pass sums every bucket's records in LDS and adds
// the sums to the workspace.
#include <cstdlib>

#include "common.h"
#include "internal.h"
#include "symm_layout.h"

namespace spsyrk {
namespace {

constexpr int kTileS = 4096;              // entries per workgroup (16 per thread with one column)
constexpr int kWinS = 1024;               // rows held in LDS

__device__ inline int64_t last_leq_s(const int64_t* a, int64_t lo, int64_t hi, int64_t x) {
    // largest i in [lo, hi] with a[i] <= x (a non-decreasing, a[lo] <= x)
    while (lo < hi) {
        const int64_t mid = (lo + hi + 1) >> 1;
        if (a[mid] <= x)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

// Columns [q0, q0 + KB) of X and of the workspace W (m x k, row-major).  The
// workgroup's tile is split into kBlock / KB groups of KB lanes; a group
// walks a stretch of consecutive entries and its lane q takes column q0 + q,
// so the KB columns of an entry are gathered, and added to, as one
// contiguous run of a row of X and of W.
template <typename V, typename XT, int KB>
__global__ __launch_bounds__(kBlock) void symm_kernel(const int64_t* __restrict__ rp, int64_t m, int64_t nnz,
                                                      const int32_t* __restrict__ ci, const V* __restrict__ cv,
                                                      const int64_t* __restrict__ trow, const XT* __restrict__ x,
                                                      int64_t ldx, int64_t k, int64_t q0, double* __restrict__ w) {
    constexpr int kGroups = kBlock / KB;
    constexpr int kPerG = kTileS / kGroups;  // entries per group
    constexpr int kBatch = 8;                // entries whose loads are issued together
    static_assert(kPerG % kBatch == 0, "whole batches");
    __shared__ int64_t win[kWinS + 1];
    __shared__ int64_t bounds[2];
    const int64_t e0 = int64_t(blockIdx.x) * kTileS;
    const int64_t e1 = min(nnz, e0 + kTileS);
    if (threadIdx.x == 0) {
        const int64_t lo = trow[blockIdx.x];
        bounds[0] = lo;
        bounds[1] = e1 < nnz ? trow[blockIdx.x + 1] : last_leq_s(rp, lo, m, e1 - 1);
    }
    __syncthreads();
    const int64_t rlo = bounds[0], rhi = bounds[1];
    const bool staged = rhi - rlo + 1 <= kWinS;
    if (staged)
        for (int64_t t = threadIdx.x; t <= rhi - rlo + 1 && rlo + t <= m; t += kBlock) win[t] = rp[rlo + t];
    __syncthreads();
    const int g = threadIdx.x / KB, q = threadIdx.x % KB;
    const int64_t a = e0 + int64_t(g) * kPerG;
    const int64_t b = min(e1, a + kPerG);
    if (a >= b) return;
    int64_t r = staged ? rlo + last_leq_s(win, 0, rhi - rlo, a) : last_leq_s(rp, rlo, rhi, a);
    int64_t rend = staged ? win[r - rlo + 1] : rp[r + 1];
    double xi = double(x[r * ldx + q0 + q]);
    double dot = 0.0;
    for (int64_t a0 = a; a0 < b; a0 += kBatch) {
        int32_t cj[kBatch];
        double cvv[kBatch], xj[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const bool in = a0 + u < b;
            cj[u] = in ? ci[a0 + u] : 0;
            cvv[u] = in ? double(cv[a0 + u]) : 0.0;
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) xj[u] = a0 + u < b ? double(x[int64_t(cj[u]) * ldx + q0 + q]) : 0.0;
        for (int u = 0; u < kBatch; ++u) {
            const int64_t e = a0 + u;
            if (e >= b) break;
            if (e >= rend) {
                // the row ends inside the stretch: add its row term
                atomicAdd(&w[r * k + q0 + q], dot);
                do {  // the row of e (empty rows add nothing)
                    ++r;
                    rend = staged && r <= rhi ? win[r - rlo + 1] : rp[r + 1];
                } while (rend <= e);
                xi = double(x[r * ldx + q0 + q]);
                dot = 0.0;
            }
            const int64_t j = cj[u];
            dot += cvv[u] * xj[u];
            if (j != r) atomicAdd(&w[j * k + q0 + q], cvv[u] * xi);
        }
    }
    atomicAdd(&w[r * k + q0 + q], dot);
}

// Rows of Y per bucket: 2^BITS, BITS from 12 to 14 picked so that there are
// at most 256 buckets where possible (a workgroup's records of one bucket
// then form stretches of 256 or more); at most kMaxBkts buckets.
constexpr int kMaxBkts = kSymmMaxBuckets;
constexpr int kSub = 32;                        // tiles of kTileS entries per bucketing workgroup
constexpr int64_t kPart = 65536;                // records summed per workgroup

// Entries [blk * kSub * kTileS, +kSub * kTileS) of workgroup blk: the count of
// its entries per bucket of their column, cnt[bucket * nblk + blk].  Every
// entry counts, the diagonal too (its record holds zero).
template <int BITS>
__global__ __launch_bounds__(kBlock) void bucket_count(const int32_t* __restrict__ ci, int64_t nnz, int nbk,
                                                       int64_t nblk, int64_t* __restrict__ cnt) {
    __shared__ uint32_t h[kMaxBkts];
    for (int b = threadIdx.x; b < nbk; b += kBlock) h[b] = 0;
    __syncthreads();
    const int64_t e0 = int64_t(blockIdx.x) * kSub * kTileS;
    const int64_t e1 = min(nnz, e0 + int64_t(kSub) * kTileS);
    for (int64_t e = e0 + threadIdx.x; e < e1; e += kBlock) atomicAdd(&h[ci[e] >> BITS], 1u);
    __syncthreads();
    for (int b = threadIdx.x; b < nbk; b += kBlock) cnt[int64_t(b) * nblk + blockIdx.x] = h[b];
}

// The row pass for one column with the transposed terms written as records:
// kSub tiles of kTileS entries per workgroup, one thread per stretch of
// entries as in symm_kernel.  boff: the exclusive scan of bucket_count's
// counts, so that this workgroup's records of bucket b go to
// [boff[b * nblk + blk], ...), claimed through LDS cursors.
template <typename V, typename XT, int BITS>
__global__ __launch_bounds__(kBlock) void symm_records(const int64_t* __restrict__ rp, int64_t m, int64_t nnz,
                                                       const int32_t* __restrict__ ci, const V* __restrict__ cv,
                                                       const int64_t* __restrict__ trow, const XT* __restrict__ x,
                                                       int64_t ldx, double* __restrict__ w,
                                                       const int64_t* __restrict__ boff, int nbk, int64_t nblk,
                                                       uint16_t* __restrict__ rj, double* __restrict__ rv) {
    constexpr int kPerG = kTileS / kBlock;  // entries per thread and tile
    constexpr int kBatch = 8;
    static_assert(kPerG % kBatch == 0, "whole batches");
    __shared__ int64_t cur[kMaxBkts];
    __shared__ int64_t win[kWinS + 1];
    __shared__ int64_t bounds[2];
    for (int b = threadIdx.x; b < nbk; b += kBlock) cur[b] = boff[int64_t(b) * nblk + blockIdx.x];
    const int64_t ntiles = (nnz + kTileS - 1) / kTileS;
    for (int sub = 0; sub < kSub; ++sub) {
        const int64_t tile = int64_t(blockIdx.x) * kSub + sub;
        if (tile >= ntiles) break;  // uniform over the workgroup
        const int64_t e0 = tile * kTileS;
        const int64_t e1 = min(nnz, e0 + kTileS);
        __syncthreads();  // the previous tile's window is spent; the cursors are set
        if (threadIdx.x == 0) {
            const int64_t lo = trow[tile];
            bounds[0] = lo;
            bounds[1] = e1 < nnz ? trow[tile + 1] : last_leq_s(rp, lo, m, e1 - 1);
        }
        __syncthreads();
        const int64_t rlo = bounds[0], rhi = bounds[1];
        const bool staged = rhi - rlo + 1 <= kWinS;
        if (staged)
            for (int64_t t = threadIdx.x; t <= rhi - rlo + 1 && rlo + t <= m; t += kBlock) win[t] = rp[rlo + t];
        __syncthreads();
        const int64_t a = e0 + int64_t(threadIdx.x) * kPerG;
        const int64_t b = min(e1, a + kPerG);
        if (a >= b) continue;
        int64_t r = staged ? rlo + last_leq_s(win, 0, rhi - rlo, a) : last_leq_s(rp, rlo, rhi, a);
        int64_t rend = staged ? win[r - rlo + 1] : rp[r + 1];
        double xi = double(x[r * ldx]);
        double dot = 0.0;
        for (int64_t a0 = a; a0 < b; a0 += kBatch) {
            int32_t cj[kBatch];
            double cvv[kBatch], xj[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const bool in = a0 + u < b;
                cj[u] = in ? ci[a0 + u] : 0;
                cvv[u] = in ? double(cv[a0 + u]) : 0.0;
            }
#pragma unroll
            for (int u = 0; u < kBatch; ++u) xj[u] = a0 + u < b ? double(x[int64_t(cj[u]) * ldx]) : 0.0;
            for (int u = 0; u < kBatch; ++u) {
                const int64_t e = a0 + u;
                if (e >= b) break;
                if (e >= rend) {
                    atomicAdd(&w[r], dot);
                    do {
                        ++r;
                        rend = staged && r <= rhi ? win[r - rlo + 1] : rp[r + 1];
                    } while (rend <= e);
                    xi = double(x[r * ldx]);
                    dot = 0.0;
                }
                const int64_t j = cj[u];
                dot += cvv[u] * xj[u];
                const int64_t slot = atomicAdd(reinterpret_cast<unsigned long long*>(&cur[j >> BITS]), 1ull);
                rj[slot] = uint16_t(j & ((1 << BITS) - 1));
                rv[slot] = j != r ? cvv[u] * xi : 0.0;
            }
        }
        atomicAdd(&w[r], dot);
    }
}

// Records [p * kPart, +kPart) of the bucket-major array: each bucket's part
// summed in LDS, then added to its rows of the workspace.
template <int BITS>
__global__ __launch_bounds__(kBlock) void bucket_sum(const int64_t* __restrict__ boff, int nbk, int64_t nblk,
                                                     int64_t nrec, const uint16_t* __restrict__ rj,
                                                     const double* __restrict__ rv, double* __restrict__ w) {
    constexpr int kBkt = 1 << BITS;
    __shared__ double acc[kBkt];
    __shared__ int first;
    const int64_t s0 = int64_t(blockIdx.x) * kPart, s1 = min(nrec, s0 + kPart);
    if (threadIdx.x == 0) {
        int lo = 0, hi = nbk - 1;  // the last bucket starting at or before s0
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (boff[int64_t(mid) * nblk] <= s0)
                lo = mid;
            else
                hi = mid - 1;
        }
        first = lo;
    }
    __syncthreads();
    for (int b = first; b < nbk; ++b) {
        const int64_t bs = boff[int64_t(b) * nblk];
        if (bs >= s1) break;  // uniform over the workgroup
        const int64_t be = b + 1 < nbk ? boff[int64_t(b + 1) * nblk] : nrec;
        const int64_t lo = max(s0, bs), hi = min(s1, be);
        if (lo >= hi) continue;
        for (int t = threadIdx.x; t < kBkt; t += kBlock) acc[t] = 0.0;
        __syncthreads();
        constexpr int kU = 4;
        for (int64_t s = lo + threadIdx.x; s < hi; s += int64_t(kBlock) * kU) {
            uint16_t jj[kU];
            double vv[kU];
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int64_t q = s + int64_t(u) * kBlock;
                jj[u] = q < hi ? rj[q] : 0;
                vv[u] = q < hi ? rv[q] : 0.0;
            }
#pragma unroll
            for (int u = 0; u < kU; ++u)
                if (s + int64_t(u) * kBlock < hi) atomicAdd(&acc[jj[u]], vv[u]);
        }
        __syncthreads();
        const int64_t r0 = int64_t(b) << BITS;
        for (int t = threadIdx.x; t < kBkt; t += kBlock)
            if (acc[t] != 0.0) atomicAdd(&w[r0 + t], acc[t]);
        __syncthreads();
    }
}

// ---- split path (one column, past 2^21 rows): the transposed terms as
// records (row in its range, value) grouped by ranges of 2^bits rows of Y,
// every tile's records sorted by range in LDS and written as one contiguous
// run per range; then one workgroup per range sums its records in LDS and
// adds the sums to its rows of the workspace.

constexpr int kSplitRows = 1 << 14;  // rows per range at most (the LDS accumulator)
// threads of a record-writing workgroup: its LDS (about 72 KiB: the tile's
// records sorted by range) lets two share a compute unit, so the workgroup
// is large enough for four wavefronts per SIMD to hide the gathers of X (256
// threads measure 10% slower, 1024 25% slower; tiles of 2048 entries with
// three workgroups per compute unit 15% slower: shorter runs per range)
constexpr int kSplitThreads = 512;

// Entries [blk * kSub * kTileS, +kSub * kTileS) of workgroup blk: its entries
// per range of their column, cnt[range * nblk + blk] (every entry, the
// diagonal too: its record holds zero).
__global__ __launch_bounds__(kBlock) void split_count(const int32_t* __restrict__ ci, int64_t nnz, int bits, int nr,
                                                      int64_t nblk, int64_t* __restrict__ cnt) {
    __shared__ uint32_t h[kSymmSplitMax];
    for (int b = threadIdx.x; b < nr; b += kBlock) h[b] = 0;
    __syncthreads();
    const int64_t e0 = int64_t(blockIdx.x) * kSub * kTileS;
    const int64_t e1 = min(nnz, e0 + int64_t(kSub) * kTileS);
    for (int64_t e = e0 + threadIdx.x; e < e1; e += kBlock) atomicAdd(&h[ci[e] >> bits], 1u);
    __syncthreads();
    for (int b = threadIdx.x; b < nr; b += kBlock) cnt[int64_t(b) * nblk + blockIdx.x] = h[b];
}

// The row pass for one column, kSub tiles of kTileS entries per workgroup,
// one thread per stretch of kTileS / kBlock entries as in symm_kernel; the
// row term is added per row stretch.  Each tile's transposed terms are
// counted per range, placed in LDS range by range, and written out as one
// contiguous run per range at the range's cursor of this workgroup (boff:
// exclusive scan of split_count's counts).
template <typename V, typename XT>
__global__ __launch_bounds__(kSplitThreads) void split_records(const int64_t* __restrict__ rp, int64_t m, int64_t nnz,
                                                        const int32_t* __restrict__ ci, const V* __restrict__ cv,
                                                        const int64_t* __restrict__ trow, const XT* __restrict__ x,
                                                        int64_t ldx, double* __restrict__ w,
                                                        const int64_t* __restrict__ boff, int bits, int nr,
                                                        int64_t nblk, uint16_t* __restrict__ rj,
                                                        double* __restrict__ rv) {
    constexpr int kPerG = kTileS / kSplitThreads;  // entries per thread
    constexpr int kBatch = kPerG < 8 ? kPerG : 8;
    static_assert(kPerG % kBatch == 0, "whole batches");
    __shared__ int64_t cur[kSymmSplitMax];   // next record of each range for this workgroup
    __shared__ uint32_t th[kSymmSplitMax];   // the tile's records per range, then their LDS start
    __shared__ uint32_t tc[kSymmSplitMax];   // placement cursors inside the tile
    __shared__ uint32_t wt[kSplitThreads / kWave];
    __shared__ uint16_t sj[kTileS];
    __shared__ uint16_t sb[kTileS];
    __shared__ double sv[kTileS];
    __shared__ int64_t win[kWinS + 1];
    __shared__ int64_t bounds[2];
    for (int b = threadIdx.x; b < nr; b += kSplitThreads) {
        cur[b] = boff[int64_t(b) * nblk + blockIdx.x];
        th[b] = 0;
        tc[b] = 0;
    }
    const uint32_t lmask = (1u << bits) - 1u;
    const int64_t ntiles = (nnz + kTileS - 1) / kTileS;
    for (int sub = 0; sub < kSub; ++sub) {
        const int64_t tile = int64_t(blockIdx.x) * kSub + sub;
        if (tile >= ntiles) break;  // uniform over the workgroup
        const int64_t e0 = tile * kTileS;
        const int64_t e1 = min(nnz, e0 + kTileS);
        __syncthreads();  // the previous tile is written; counters are reset
        if (threadIdx.x == 0) {
            const int64_t lo = trow[tile];
            bounds[0] = lo;
            bounds[1] = e1 < nnz ? trow[tile + 1] : last_leq_s(rp, lo, m, e1 - 1);
        }
        __syncthreads();
        const int64_t rlo = bounds[0], rhi = bounds[1];
        const bool staged = rhi - rlo + 1 <= kWinS;
        if (staged)
            for (int64_t t = threadIdx.x; t <= rhi - rlo + 1 && rlo + t <= m; t += kSplitThreads) win[t] = rp[rlo + t];
        __syncthreads();
        const int64_t a = e0 + int64_t(threadIdx.x) * kPerG;
        const int64_t b = min(e1, a + kPerG);
        uint32_t rb[kPerG];  // range (high bits) and row in range (low 16 bits) of each term
        double tv[kPerG];
#pragma unroll
        for (int u = 0; u < kPerG; ++u) {
            rb[u] = 0xffffffffu;
            tv[u] = 0.0;
        }
        if (a < b) {
            int64_t r = staged ? rlo + last_leq_s(win, 0, rhi - rlo, a) : last_leq_s(rp, rlo, rhi, a);
            int64_t rend = staged ? win[r - rlo + 1] : rp[r + 1];
            double xi = double(x[r * ldx]);
            double dot = 0.0;
#pragma unroll
            for (int h = 0; h < kPerG; h += kBatch) {
                const int64_t a0 = a + h;
                int32_t cj[kBatch];
                double cvv[kBatch], xj[kBatch];
#pragma unroll
                for (int u = 0; u < kBatch; ++u) {
                    const bool in = a0 + u < b;
                    cj[u] = in ? ci[a0 + u] : 0;
                    cvv[u] = in ? double(cv[a0 + u]) : 0.0;
                }
#pragma unroll
                for (int u = 0; u < kBatch; ++u) xj[u] = a0 + u < b ? double(x[int64_t(cj[u]) * ldx]) : 0.0;
#pragma unroll
                for (int u = 0; u < kBatch; ++u) {
                    const int64_t e = a0 + u;
                    if (e < b) {
                        if (e >= rend) {
                            atomicAdd(&w[r], dot);
                            do {
                                ++r;
                                rend = staged && r <= rhi ? win[r - rlo + 1] : rp[r + 1];
                            } while (rend <= e);
                            xi = double(x[r * ldx]);
                            dot = 0.0;
                        }
                        const uint32_t j = uint32_t(cj[u]);
                        dot += cvv[u] * xj[u];
                        rb[h + u] = ((j >> bits) << 16) | (j & lmask);
                        tv[h + u] = int64_t(j) != r ? cvv[u] * xi : 0.0;
                    }
                }
            }
            atomicAdd(&w[r], dot);
        }
        // the tile's records per range, their LDS places, then their runs
#pragma unroll
        for (int u = 0; u < kPerG; ++u)
            if (rb[u] != 0xffffffffu) atomicAdd(&th[rb[u] >> 16], 1u);
        __syncthreads();
        block_exclusive_scan_array<uint32_t, kSplitThreads>(th, nr, wt);  // th: start of each range's run in LDS
        __syncthreads();
#pragma unroll
        for (int u = 0; u < kPerG; ++u) {
            if (rb[u] == 0xffffffffu) continue;
            const uint32_t g = rb[u] >> 16;
            const uint32_t q = th[g] + atomicAdd(&tc[g], 1u);
            sj[q] = uint16_t(rb[u] & 0xffffu);
            sb[q] = uint16_t(g);
            sv[q] = tv[u];
        }
        __syncthreads();
        const int tn = int(e1 - e0);
        for (int q = threadIdx.x; q < tn; q += kSplitThreads) {
            const uint32_t g = sb[q];
            const int64_t dst = cur[g] + int64_t(q - int(th[g]));
            rj[dst] = sj[q];
            rv[dst] = sv[q];
        }
        __syncthreads();
        for (int g = threadIdx.x; g < nr; g += kSplitThreads) {
            cur[g] += tc[g];
            th[g] = 0;
            tc[g] = 0;
        }
    }
}

// Range blockIdx.x: its records (every workgroup's run, contiguous in the
// range-major array) summed in LDS, then added to its rows of the workspace
// (no other workgroup touches them).
__global__ __launch_bounds__(kBlock) void split_apply(const int64_t* __restrict__ boff, int nr, int64_t nblk,
                                                      int64_t nrec, int bits, int64_t m,
                                                      const uint16_t* __restrict__ rj,
                                                      const double* __restrict__ rv, double* __restrict__ w) {
    __shared__ double acc[kSplitRows];
    const int rg = blockIdx.x;
    const int rows = int(min(int64_t(1) << bits, m - (int64_t(rg) << bits)));
    for (int t = threadIdx.x; t < rows; t += kBlock) acc[t] = 0.0;
    __syncthreads();
    const int64_t s0 = boff[int64_t(rg) * nblk];
    const int64_t s1 = rg + 1 < nr ? boff[int64_t(rg + 1) * nblk] : nrec;
    constexpr int kU = 4;
    for (int64_t q0 = s0 + threadIdx.x; q0 < s1; q0 += int64_t(kBlock) * kU) {
        uint32_t jj[kU];
        double vv[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int64_t q = q0 + int64_t(u) * kBlock;
            jj[u] = q < s1 ? rj[q] : 0u;
            vv[u] = q < s1 ? rv[q] : 0.0;
        }
#pragma unroll
        for (int u = 0; u < kU; ++u)
            if (vv[u] != 0.0) atomicAdd(&acc[jj[u]], vv[u]);
    }
    __syncthreads();
    double* __restrict__ wr = w + (int64_t(rg) << bits);
    for (int t = threadIdx.x; t < rows; t += kBlock) wr[t] += acc[t];
}

__global__ __launch_bounds__(kBlock) void zero_f64(double* __restrict__ p, int64_t n) {
    for (int64_t i = int64_t(blockIdx.x) * kBlock + threadIdx.x; i < n; i += int64_t(gridDim.x) * kBlock) p[i] = 0.0;
}

template <typename XT>
__global__ __launch_bounds__(kBlock) void store_y(const double* __restrict__ w, int64_t m, int64_t k,
                                                  XT* __restrict__ y, int64_t ldy) {
    for (int64_t i = int64_t(blockIdx.x) * kBlock + threadIdx.x; i < m * k; i += int64_t(gridDim.x) * kBlock) {
        const int64_t r = i / k, q = i - r * k;
        y[r * ldy + q] = XT(w[i]);
    }
}

unsigned grid_for(int64_t n) {
    int64_t g = (n + kBlock - 1) / kBlock;
    return unsigned(g < 1 ? 1 : (g > 65536 ? 65536 : g));
}

template <typename V, typename XT>
void launch_symm(const DevCsr& C, const XT* x, int64_t ldx, int64_t k, double* w, const int64_t* trow,
                 hipStream_t s) {
    const unsigned nb = unsigned((C.nnz + kTileS - 1) / kTileS);
    const V* cv = static_cast<const V*>(C.v);
    for (int64_t q0 = 0; q0 < k;) {
        const int64_t left = k - q0;
        if (left >= 8) {
            symm_kernel<V, XT, 8><<<nb, kBlock, 0, s>>>(C.rp, C.m, C.nnz, C.ci, cv, trow, x, ldx, k, q0, w);
            q0 += 8;
        } else if (left >= 4) {
            symm_kernel<V, XT, 4><<<nb, kBlock, 0, s>>>(C.rp, C.m, C.nnz, C.ci, cv, trow, x, ldx, k, q0, w);
            q0 += 4;
        } else if (left >= 2) {
            symm_kernel<V, XT, 2><<<nb, kBlock, 0, s>>>(C.rp, C.m, C.nnz, C.ci, cv, trow, x, ldx, k, q0, w);
            q0 += 2;
        } else {
            symm_kernel<V, XT, 1><<<nb, kBlock, 0, s>>>(C.rp, C.m, C.nnz, C.ci, cv, trow, x, ldx, k, q0, w);
            q0 += 1;
        }
    }
}

size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

// The transposed term of a single column goes through buckets when its
// workspace outgrows one XCD's L2 (4 MiB: 2^19 rows), where random atomic adds
// miss, up to 2^21 rows: past that the buckets are too many for a workgroup's
// stretches of records to fill whole cache lines, and the scattered record
// writes cost as much as the atomic adds.  SPSYRK_SYMM_BUCKETS (read at every
// call) = 0 turns buckets off; = 1 takes them for every single column of up to
// 2^24 rows; = 12, 13 or 14 does the same with buckets of 2^12, 2^13 or 2^14
// rows, raised where needed to keep the buckets at most kSymmMaxBuckets.
int forced_bits() {
    const char* e = std::getenv("SPSYRK_SYMM_BUCKETS");
    if (!e) return -1;
    const int v = std::atoi(e);
    return v == 0 || v == 1 || (v >= 12 && v <= 14) ? v : -1;
}

bool bucketed(int64_t m, int64_t k, int64_t nnz) { return symm_bucketed(m, k, nnz, forced_bits()); }

// SPSYRK_SYMM_SPLIT (read at every call): 0 never splits, 1 splits every
// single column; unset, single columns past 2^21 rows are split.
// SPSYRK_SYMM_SPLIT_BITS: rows per range 2^bits instead of 2^18 (tests use
// it to get several ranges out of small matrices).
int forced_split() {
    const char* e = std::getenv("SPSYRK_SYMM_SPLIT");
    if (!e) return -1;
    return e[0] == '0' ? 0 : (e[0] == '1' ? 1 : -1);
}

int forced_split_bits() {
    const char* e = std::getenv("SPSYRK_SYMM_SPLIT_BITS");
    return e ? std::atoi(e) : 0;
}

struct SplitLayout {
    int bits;
    int nr;
    int64_t nblk;
    size_t boff, stmp, rj, rv, end;  // byte offsets after the workspace and the tile rows
};

struct BucketLayout {
    int bits;
    int nbk;
    int64_t nblk;
    size_t boff, stmp, rj, rv, end;  // byte offsets after the workspace and the tile rows
};

BucketLayout bucket_layout(int64_t m, int64_t nnz, size_t base) {
    BucketLayout L;
    L.bits = symm_bucket_bits(m, forced_bits());
    L.nbk = symm_bucket_count(m, L.bits);  // <= kMaxBkts whenever bucketed() holds
    const int64_t ntiles = (nnz + kTileS - 1) / kTileS;
    L.nblk = (ntiles + kSub - 1) / kSub;
    const int64_t ncnt = int64_t(L.nbk) * L.nblk;
    L.boff = base;
    L.stmp = L.boff + align256(size_t(ncnt) * sizeof(int64_t));
    L.rj = L.stmp + align256(scan_tmp_bytes(ncnt));
    L.rv = L.rj + align256(size_t(nnz) * sizeof(uint16_t));
    L.end = L.rv + size_t(nnz) * sizeof(double);
    return L;
}

size_t symm_base_bytes(int64_t m, int64_t k, int64_t nnz) {
    return align256(size_t(m) * size_t(k) * sizeof(double)) +
           align256(size_t((nnz + kTileS - 1) / kTileS + 1) * sizeof(int64_t));
}

SplitLayout split_layout(int64_t m, int64_t nnz, size_t base) {
    SplitLayout L;
    L.bits = symm_split_bits(m, forced_split_bits());
    L.nr = int((m + (int64_t(1) << L.bits) - 1) >> L.bits);
    const int64_t ntiles = (nnz + kTileS - 1) / kTileS;
    L.nblk = (ntiles + kSub - 1) / kSub;
    const int64_t ncnt = int64_t(L.nr) * L.nblk;
    L.boff = base;
    L.stmp = L.boff + align256(size_t(ncnt) * sizeof(int64_t));
    L.rj = L.stmp + align256(scan_tmp_bytes(ncnt));
    L.rv = L.rj + align256(size_t(nnz) * sizeof(uint16_t));
    L.end = L.rv + size_t(nnz) * sizeof(double);
    return L;
}

template <typename V, typename XT>
void launch_split(const DevCsr& C, const XT* x, int64_t ldx, double* w, const int64_t* trow, char* tmp,
                  const SplitLayout& L, hipStream_t s) {
    int64_t* boff = reinterpret_cast<int64_t*>(tmp + L.boff);
    uint16_t* rj = reinterpret_cast<uint16_t*>(tmp + L.rj);
    double* rv = reinterpret_cast<double*>(tmp + L.rv);
    split_count<<<unsigned(L.nblk), kBlock, 0, s>>>(C.ci, C.nnz, L.bits, L.nr, L.nblk, boff);
    scan_i64(boff, boff, int64_t(L.nr) * L.nblk, nullptr, tmp + L.stmp, s);
    split_records<V, XT><<<unsigned(L.nblk), kSplitThreads, 0, s>>>(C.rp, C.m, C.nnz, C.ci, static_cast<const V*>(C.v), trow,
                                                             x, ldx, w, boff, L.bits, L.nr, L.nblk, rj, rv);
    split_apply<<<unsigned(L.nr), kBlock, 0, s>>>(boff, L.nr, L.nblk, C.nnz, L.bits, C.m, rj, rv, w);
}

template <typename V, typename XT, int BITS>
void launch_bucketed_bits(const DevCsr& C, const XT* x, int64_t ldx, double* w, const int64_t* trow, char* tmp,
                          const BucketLayout& L, hipStream_t s) {
    int64_t* boff = reinterpret_cast<int64_t*>(tmp + L.boff);
    uint16_t* rj = reinterpret_cast<uint16_t*>(tmp + L.rj);
    double* rv = reinterpret_cast<double*>(tmp + L.rv);
    bucket_count<BITS><<<unsigned(L.nblk), kBlock, 0, s>>>(C.ci, C.nnz, L.nbk, L.nblk, boff);
    scan_i64(boff, boff, int64_t(L.nbk) * L.nblk, nullptr, tmp + L.stmp, s);
    symm_records<V, XT, BITS><<<unsigned(L.nblk), kBlock, 0, s>>>(C.rp, C.m, C.nnz, C.ci,
                                                                   static_cast<const V*>(C.v), trow, x, ldx, w, boff,
                                                                   L.nbk, L.nblk, rj, rv);
    const unsigned np = unsigned((C.nnz + kPart - 1) / kPart);
    bucket_sum<BITS><<<np, kBlock, 0, s>>>(boff, L.nbk, L.nblk, C.nnz, rj, rv, w);
}

template <typename V, typename XT>
void launch_bucketed(const DevCsr& C, const XT* x, int64_t ldx, double* w, const int64_t* trow, char* tmp,
                     const BucketLayout& L, hipStream_t s) {
    switch (L.bits) {
        case 12: launch_bucketed_bits<V, XT, 12>(C, x, ldx, w, trow, tmp, L, s); break;
        case 13: launch_bucketed_bits<V, XT, 13>(C, x, ldx, w, trow, tmp, L, s); break;
        default: launch_bucketed_bits<V, XT, 14>(C, x, ldx, w, trow, tmp, L, s); break;
    }
}

}  // namespace

int symm_mode(int64_t m, int64_t k, int64_t nnz) {
    if (bucketed(m, k, nnz)) return kSymmBuckets;
    if (symm_split(m, k, nnz, forced_split(), forced_split_bits())) return kSymmSplit;
    return kSymmAtomics;
}

size_t symm_tmp_bytes(int64_t m, int64_t k, int64_t nnz, int mode) {
    const size_t base = symm_base_bytes(m, k, nnz);
    if (mode == kSymmBuckets) return bucket_layout(m, nnz, base).end;
    if (mode == kSymmSplit) return split_layout(m, nnz, base).end;
    return base;
}

void symm_product(const DevCsr& C, int sr, const void* x, int64_t ldx, int64_t k, void* y, int64_t ldy, void* tmp,
                  int mode, hipStream_t s) {
    double* w = static_cast<double*>(tmp);
    int64_t* trow = reinterpret_cast<int64_t*>(static_cast<char*>(tmp) + align256(size_t(C.m) * size_t(k) * sizeof(double)));
    zero_f64<<<grid_for(C.m * k), kBlock, 0, s>>>(w, C.m * k);
    if (mode == kSymmSplit && C.nnz > 0) {
        tile_first_rows(C.rp, C.m, kTileS, trow, s);
        const SplitLayout L = split_layout(C.m, C.nnz, symm_base_bytes(C.m, k, C.nnz));
        char* t = static_cast<char*>(tmp);
        switch (sr) {
            case kF64: launch_split<double, double>(C, static_cast<const double*>(x), ldx, w, trow, t, L, s); break;
            case kCount: launch_split<int32_t, double>(C, static_cast<const double*>(x), ldx, w, trow, t, L, s); break;
            default: launch_split<float, float>(C, static_cast<const float*>(x), ldx, w, trow, t, L, s); break;
        }
    } else if (mode == kSymmBuckets && C.nnz > 0) {
        tile_first_rows(C.rp, C.m, kTileS, trow, s);
        const BucketLayout L = bucket_layout(C.m, C.nnz, symm_base_bytes(C.m, k, C.nnz));
        char* t = static_cast<char*>(tmp);
        switch (sr) {
            case kF64: launch_bucketed<double, double>(C, static_cast<const double*>(x), ldx, w, trow, t, L, s); break;
            case kCount: launch_bucketed<int32_t, double>(C, static_cast<const double*>(x), ldx, w, trow, t, L, s); break;
            default: launch_bucketed<float, float>(C, static_cast<const float*>(x), ldx, w, trow, t, L, s); break;
        }
    } else if (C.nnz > 0) {
        tile_first_rows(C.rp, C.m, kTileS, trow, s);
        switch (sr) {
            case kF64: launch_symm<double, double>(C, static_cast<const double*>(x), ldx, k, w, trow, s); break;
            case kF32: launch_symm<float, float>(C, static_cast<const float*>(x), ldx, k, w, trow, s); break;
            case kCount: launch_symm<int32_t, double>(C, static_cast<const double*>(x), ldx, k, w, trow, s); break;
            default: launch_symm<float, float>(C, static_cast<const float*>(x), ldx, k, w, trow, s); break;
        }
    }
    if (sr == kF64 || sr == kCount)
        store_y<double><<<grid_for(C.m * k), kBlock, 0, s>>>(w, C.m, k, static_cast<double*>(y), ldy);
    else
        store_y<float><<<grid_for(C.m * k), kBlock, 0, s>>>(w, C.m, k, static_cast<float*>(y), ldy);
}

}  // namespace spsyrk
