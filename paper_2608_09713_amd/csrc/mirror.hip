// Symmetric completion C = C_L + C_L^T - D (Eq. (spmv)) of a stored lower
// part.  Row i of C is row i of C_L followed by column i of the strict lower
// part in ascending row order.  The lower rows are copied in place; the
// strict lower part is transposed by a stable sort of (column, row, value)
// records by column, in column slabs that bound the record buffers, and each
// sorted record is dropped at its place in the full row.
#include "common.h"
#include "internal.h"

namespace spsyrk {
namespace {

constexpr int kTileE = 4096;
constexpr int kWin = 4096;

// Row of each entry of a tile [e0, e1): staged window of row_ptr, or a
// direct search when the tile spans too many (empty) rows.
struct RowFinder {
    const int64_t* rp;
    int64_t rlo, rhi;
    bool staged;
    const int64_t* win;
    __device__ int64_t row_of(int64_t e) const {
        if (staged) {
            int lo = 0, hi = int(rhi - rlo);
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (win[mid] <= e)
                    lo = mid;
                else
                    hi = mid - 1;
            }
            return rlo + lo;
        }
        int64_t lo = rlo, hi = rhi;
        while (lo < hi) {
            const int64_t mid = (lo + hi + 1) >> 1;
            if (rp[mid] <= e)
                lo = mid;
            else
                hi = mid - 1;
        }
        return lo;
    }
};

__device__ inline int64_t last_row_leq(const int64_t* rp, int64_t m, int64_t e) {
    int64_t lo = 0, hi = m;
    while (lo < hi) {
        const int64_t mid = (lo + hi + 1) >> 1;
        if (rp[mid] <= e)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

__device__ inline RowFinder make_finder(const int64_t* rp, int64_t m, int64_t e0, int64_t e1, int64_t* win,
                                        int64_t* bounds) {
    if (threadIdx.x == 0) {
        bounds[0] = last_row_leq(rp, m, e0);
        bounds[1] = last_row_leq(rp, m, e1 - 1);
    }
    __syncthreads();
    RowFinder f{rp, bounds[0], bounds[1], false, win};
    const int64_t nwin = f.rhi - f.rlo + 2;
    if (nwin <= kWin + 1) {
        for (int64_t k = threadIdx.x; k < nwin; k += kBlock) win[k] = rp[f.rlo + k];
        f.staged = true;
    }
    __syncthreads();
    return f;
}

// Strict-lower entries per column (32-bit counters; a column holds fewer than
// 2^31 entries).  Every thread walks kPerC contiguous entries row by row, so
// the diagonal (the last entry of a row, col == row) is recognised without a
// search per entry.
constexpr int kPerC = 16;
constexpr int kTileC = kBlock * kPerC;

__global__ __launch_bounds__(kBlock) void count_transposed(const int64_t* __restrict__ rp,
                                                           const int32_t* __restrict__ ci, int64_t m, int64_t nnz,
                                                           uint32_t* __restrict__ cnt) {
    __shared__ int64_t win[kWin + 1];
    __shared__ int64_t bounds[2];
    const int64_t e0 = int64_t(blockIdx.x) * kTileC;
    const int64_t e1 = min(nnz, e0 + kTileC);
    RowFinder f = make_finder(rp, m, e0, e1, win, bounds);
    const int64_t ea = e0 + int64_t(threadIdx.x) * kPerC;
    const int64_t eb = min(e1, ea + kPerC);
    if (ea >= eb) return;
    int64_t r = f.row_of(ea);
    int64_t rend = rp[r + 1];
    for (int64_t e = ea; e < eb; ++e) {
        while (e >= rend) {  // next row (empty rows skipped)
            ++r;
            rend = rp[r + 1];
        }
        const int32_t c = ci[e];
        if (int64_t(c) < r) atomicAdd(&cnt[c], 1u);
    }
}

// full_len[i] = lower length of row i + strict-lower entries of column i;
// colcnt[i] = the latter
__global__ __launch_bounds__(kBlock) void full_lengths(const int64_t* __restrict__ rp, int64_t m,
                                                       const uint32_t* __restrict__ cnt,
                                                       int64_t* __restrict__ full_len, int64_t* __restrict__ colcnt) {
    const int64_t i = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (i >= m) return;
    full_len[i] = (rp[i + 1] - rp[i]) + int64_t(cnt[i]);
    colcnt[i] = int64_t(cnt[i]);
}

template <int VB>
__global__ __launch_bounds__(kBlock) void copy_lower(const int64_t* __restrict__ rp, const int32_t* __restrict__ ci,
                                                     const void* __restrict__ val, int64_t m, int64_t nnz,
                                                     const int64_t* __restrict__ f_rp, int32_t* __restrict__ f_ci,
                                                     void* __restrict__ f_val) {
    __shared__ int64_t win[kWin + 1];
    __shared__ int64_t bounds[2];
    const int64_t e0 = int64_t(blockIdx.x) * kTileE;
    const int64_t e1 = min(nnz, e0 + kTileE);
    RowFinder f = make_finder(rp, m, e0, e1, win, bounds);
    for (int64_t e = e0 + threadIdx.x; e < e1; e += kBlock) {
        const int64_t r = f.row_of(e);
        const int64_t p = f_rp[r] + (e - rp[r]);
        f_ci[p] = ci[e];
        if constexpr (VB == 8) static_cast<uint64_t*>(f_val)[p] = static_cast<const uint64_t*>(val)[e];
        if constexpr (VB == 4) static_cast<uint32_t*>(f_val)[p] = static_cast<const uint32_t*>(val)[e];
    }
}

__device__ inline int64_t lower_bound_i32(const int32_t* a, int64_t lo, int64_t hi, int64_t x) {
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (int64_t(a[mid]) < x)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

// entries of row r with c0 <= col < min(c1, r)
__global__ __launch_bounds__(kBlock) void slab_counts(const int64_t* __restrict__ rp, const int32_t* __restrict__ ci,
                                                      int64_t m, int64_t c0, int64_t c1, int64_t* __restrict__ cnt,
                                                      int64_t* __restrict__ lo_out) {
    const int64_t r = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (r >= m) return;
    const int64_t a = rp[r], b = rp[r + 1];
    const int64_t hi_col = min(c1, r);
    int64_t lo = a, hi = a;
    if (hi_col > c0) {
        lo = lower_bound_i32(ci, a, b, c0);
        hi = lower_bound_i32(ci, lo, b, hi_col);
    }
    cnt[r] = hi - lo;
    lo_out[r] = lo;
}

// Records [0, nrec) of a slab in row-major order: record p of row r (rows
// found in an LDS window of rec_rp) is entry row_lo[r] + (p - rec_rp[r]), so
// the slab reads only its own entries.
template <int VB>
__global__ __launch_bounds__(kBlock) void slab_extract(const int32_t* __restrict__ ci, const void* __restrict__ val,
                                                       int64_t m, int64_t c0, int64_t nrec,
                                                       const int64_t* __restrict__ rec_rp,
                                                       const int64_t* __restrict__ row_lo, uint32_t* __restrict__ rkey,
                                                       uint32_t* __restrict__ rrow, void* __restrict__ rval) {
    __shared__ int64_t win[kWin + 1];
    __shared__ int64_t bounds[2];
    const int64_t p0 = int64_t(blockIdx.x) * kTileE;
    const int64_t p1 = min(nrec, p0 + kTileE);
    RowFinder f = make_finder(rec_rp, m, p0, p1, win, bounds);
    for (int64_t p = p0 + threadIdx.x; p < p1; p += kBlock) {
        const int64_t r = f.row_of(p);
        const int64_t e = row_lo[r] + (p - rec_rp[r]);
        rkey[p] = uint32_t(int64_t(ci[e]) - c0);
        rrow[p] = uint32_t(r);
        if constexpr (VB == 8) static_cast<uint64_t*>(rval)[p] = static_cast<const uint64_t*>(val)[e];
        if constexpr (VB == 4) static_cast<uint32_t*>(rval)[p] = static_cast<const uint32_t*>(val)[e];
    }
}

template <int VB>
__global__ __launch_bounds__(kBlock) void slab_place(const int64_t* __restrict__ rp, int64_t c0, int64_t nrec,
                                                     const uint32_t* __restrict__ skey,
                                                     const uint32_t* __restrict__ srow, const void* __restrict__ sval,
                                                     const int64_t* __restrict__ cstart,
                                                     const int64_t* __restrict__ f_rp, int32_t* __restrict__ f_ci,
                                                     void* __restrict__ f_val) {
    const int64_t s = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (s >= nrec) return;
    const int64_t c = c0 + int64_t(skey[s]);
    const int64_t rank = s - (cstart[c] - cstart[c0]);
    const int64_t p = f_rp[c] + (rp[c + 1] - rp[c]) + rank;
    f_ci[p] = int32_t(srow[s]);
    if constexpr (VB == 8) static_cast<uint64_t*>(f_val)[p] = static_cast<const uint64_t*>(sval)[s];
    if constexpr (VB == 4) static_cast<uint32_t*>(f_val)[p] = static_cast<const uint32_t*>(sval)[s];
}

inline unsigned blocks_for(int64_t n, int64_t per) { return unsigned((n + per - 1) / per); }

}  // namespace

void mirror_counts(const MirrorArgs& a, uint32_t* cnt, int64_t* full_len, int64_t* colcnt, hipStream_t s) {
    if (a.m <= 0) return;
    (void)hipMemsetAsync(cnt, 0, size_t(a.m) * sizeof(uint32_t), s);
    if (a.nnz > 0)
        count_transposed<<<blocks_for(a.nnz, kTileC), kBlock, 0, s>>>(a.rp, a.ci, a.m, a.nnz, cnt);
    full_lengths<<<blocks_for(a.m, kBlock), kBlock, 0, s>>>(a.rp, a.m, cnt, full_len, colcnt);
}

void mirror_copy_lower(const MirrorArgs& a, const int64_t* f_rp, int32_t* f_ci, void* f_val, hipStream_t s) {
    const int64_t nnz = a.nnz;
    if (nnz <= 0) return;
    const unsigned nb = blocks_for(nnz, kTileE);
    if (a.vbytes == 8 && a.val)
        copy_lower<8><<<nb, kBlock, 0, s>>>(a.rp, a.ci, a.val, a.m, nnz, f_rp, f_ci, f_val);
    else if (a.vbytes == 4 && a.val)
        copy_lower<4><<<nb, kBlock, 0, s>>>(a.rp, a.ci, a.val, a.m, nnz, f_rp, f_ci, f_val);
    else
        copy_lower<0><<<nb, kBlock, 0, s>>>(a.rp, a.ci, a.val, a.m, nnz, f_rp, f_ci, f_val);
}

void mirror_slab_counts(const MirrorArgs& a, int64_t c0, int64_t c1, int64_t* row_cnt, int64_t* row_lo,
                        hipStream_t s) {
    if (a.m <= 0) return;
    slab_counts<<<blocks_for(a.m, kBlock), kBlock, 0, s>>>(a.rp, a.ci, a.m, c0, c1, row_cnt, row_lo);
}

void mirror_slab_extract(const MirrorArgs& a, int64_t c0, int64_t nrec, const int64_t* rec_rp, const int64_t* row_lo,
                         uint32_t* rkey, uint32_t* rrow, void* rval, hipStream_t s) {
    if (nrec <= 0) return;
    const unsigned nb = blocks_for(nrec, kTileE);
    if (a.vbytes == 8 && a.val)
        slab_extract<8><<<nb, kBlock, 0, s>>>(a.ci, a.val, a.m, c0, nrec, rec_rp, row_lo, rkey, rrow, rval);
    else if (a.vbytes == 4 && a.val)
        slab_extract<4><<<nb, kBlock, 0, s>>>(a.ci, a.val, a.m, c0, nrec, rec_rp, row_lo, rkey, rrow, rval);
    else
        slab_extract<0><<<nb, kBlock, 0, s>>>(a.ci, a.val, a.m, c0, nrec, rec_rp, row_lo, rkey, rrow, rval);
}

void mirror_slab_place(const MirrorArgs& a, int64_t c0, int64_t nrec, const uint32_t* skey, const uint32_t* srow,
                       const void* sval, const int64_t* cstart, const int64_t* f_rp, int32_t* f_ci, void* f_val,
                       hipStream_t s) {
    if (nrec <= 0) return;
    const unsigned nb = blocks_for(nrec, kBlock);
    if (a.vbytes == 8 && a.val)
        slab_place<8><<<nb, kBlock, 0, s>>>(a.rp, c0, nrec, skey, srow, sval, cstart, f_rp, f_ci, f_val);
    else if (a.vbytes == 4 && a.val)
        slab_place<4><<<nb, kBlock, 0, s>>>(a.rp, c0, nrec, skey, srow, sval, cstart, f_rp, f_ci, f_val);
    else
        slab_place<0><<<nb, kBlock, 0, s>>>(a.rp, c0, nrec, skey, srow, sval, cstart, f_rp, f_ci, f_val);
}

}  // namespace spsyrk
