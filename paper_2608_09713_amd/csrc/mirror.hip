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

// Rows of the tile [e0, e1) (tile t of kTileE positions, total positions in
// all): from the tile table trow (the row of every tile start; the upper
// bound may then be the row of e1, one past the tile), or by searches.
__device__ inline RowFinder make_finder(const int64_t* rp, int64_t m, int64_t e0, int64_t e1, int64_t* win,
                                        int64_t* bounds, const int64_t* trow, int64_t t, int64_t total) {
    if (threadIdx.x == 0) {
        if (trow) {
            const int64_t lo = trow[t];
            bounds[0] = lo;
            bounds[1] = e1 < total ? trow[t + 1] : last_row_leq(rp, m, e1 - 1);
        } else {
            bounds[0] = last_row_leq(rp, m, e0);
            bounds[1] = last_row_leq(rp, m, e1 - 1);
        }
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

// Every thread of a strict-lower walk takes kPerC contiguous entries row by
// row, so the diagonal (the last entry of a row, col == row) is recognised
// without a search per entry.
constexpr int kPerC = 16;
constexpr int kTileC = kBlock * kPerC;
static_assert(kTileC == kTileE, "one tile table serves the walks and the copies");

// lower rows' entries [ebeg, eend) to their places in the full rows
template <int VB>
__global__ __launch_bounds__(kBlock) void copy_lower(const int64_t* __restrict__ rp, const int32_t* __restrict__ ci,
                                                     const void* __restrict__ val, int64_t m, int64_t ebeg,
                                                     int64_t eend, const int64_t* __restrict__ trow,
                                                     const int64_t* __restrict__ f_rp, int32_t* __restrict__ f_ci,
                                                     void* __restrict__ f_val) {
    __shared__ int64_t win[kWin + 1];
    __shared__ int64_t bounds[2];
    const int64_t e0 = ebeg + int64_t(blockIdx.x) * kTileE;
    const int64_t e1 = min(eend, e0 + kTileE);
    RowFinder f = make_finder(rp, m, e0, e1, win, bounds, trow, blockIdx.x, eend);
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
        lo = c0 == 0 ? a : lower_bound_i32(ci, a, b, c0);
        if (c1 >= r)  // every column of the row below the diagonal is in the slab
            hi = (b > lo && int64_t(ci[b - 1]) == r) ? b - 1 : b;
        else
            hi = lower_bound_i32(ci, lo, b, hi_col);
    }
    cnt[r] = hi - lo;
    lo_out[r] = lo;
}

__global__ __launch_bounds__(kBlock) void slab_offsets(int64_t* __restrict__ row_lo, const int64_t* __restrict__ rec_rp,
                                                       int64_t m) {
    const int64_t r = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (r < m) row_lo[r] -= rec_rp[r];
}

// Records [0, nrec) of a slab in row-major order: record p of row r (rows
// found in an LDS window of rec_rp) is entry row_lo[r] + (p - rec_rp[r]), so
// the slab reads only its own entries.
template <int VB>
__global__ __launch_bounds__(kBlock) void slab_extract(const int32_t* __restrict__ ci, const void* __restrict__ val,
                                                       int64_t m, int64_t c0, int64_t nrec,
                                                       const int64_t* __restrict__ rec_rp,
                                                       const int64_t* __restrict__ row_lo, const int64_t* __restrict__ trow,
                                                       uint32_t* __restrict__ rkey, uint32_t* __restrict__ rrow,
                                                       void* __restrict__ rval) {
    __shared__ int64_t win[kWin + 1];
    __shared__ int64_t bounds[2];
    const int64_t p0 = int64_t(blockIdx.x) * kTileE;
    const int64_t p1 = min(nrec, p0 + kTileE);
    RowFinder f = make_finder(rec_rp, m, p0, p1, win, bounds, trow, blockIdx.x, nrec);
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
                                                     const uint32_t* __restrict__ first,
                                                     const int64_t* __restrict__ f_rp, int32_t* __restrict__ f_ci,
                                                     void* __restrict__ f_val) {
    const int64_t s = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (s >= nrec) return;
    const uint32_t k = skey[s];
    const int64_t c = c0 + int64_t(k);
    const int64_t rank = s - int64_t(first[k]);
    const int64_t p = f_rp[c] + (rp[c + 1] - rp[c]) + rank;
    f_ci[p] = int32_t(srow[s]);
    if constexpr (VB == 8) static_cast<uint64_t*>(f_val)[p] = static_cast<const uint64_t*>(sval)[s];
    if constexpr (VB == 4) static_cast<uint32_t*>(f_val)[p] = static_cast<const uint32_t*>(sval)[s];
}

// Strict-lower entries with clo <= col < clo + nb * 2^cb per bucket of 2^cb
// columns (nb <= kMirrorBins), for choosing column slabs.  Every entry of the
// lower part is counted by its column, from coalesced loads, and the diagonal
// entry of every row is taken off again (the strict lower part is the lower
// part without its diagonal).  Consecutive lanes that fall in one bucket form
// a run that its first lane adds at once, so a row's dense stretch costs one
// LDS add, not one per lane.  LDS counters per workgroup, then one global add
// per non-empty bucket.
__device__ inline void add_bucket_runs(int32_t* cnt, int b, int sign) {
    const int lane = lane_id();
    const int pb = __shfl_up(b, 1, kWave);
    const uint64_t starts = __ballot(lane == 0 || pb != b);
    if (b >= 0 && (lane == 0 || pb != b)) {
        const uint64_t after = lane == kWave - 1 ? 0 : (starts >> (lane + 1));
        const int len = after ? __ffsll((long long)after) : kWave - lane;
        atomicAdd(&cnt[b], sign * len);
    }
}

constexpr int kHistU = 4;  // 64-entry stretches per wavefront in flight

__global__ __launch_bounds__(kBlock) void coarse_hist(const int64_t* __restrict__ rp, const int32_t* __restrict__ ci,
                                                      int64_t m, int64_t nnz, int64_t clo, int cb, int nb,
                                                      unsigned long long* __restrict__ hist) {
    __shared__ int32_t cnt[kMirrorBins];
    for (int x = threadIdx.x; x < nb; x += kBlock) cnt[x] = 0;
    __syncthreads();
    const int lane = lane_id();
    const int64_t span = int64_t(nb) << cb;
    auto bucket = [&](int64_t c) -> int { return (c >= clo && c - clo < span) ? int((c - clo) >> cb) : -1; };
    const int64_t waves = int64_t(gridDim.x) * (kBlock / kWave);
    const int64_t wid = int64_t(blockIdx.x) * (kBlock / kWave) + threadIdx.x / kWave;
    // every entry, by column
    for (int64_t base = wid * (kWave * kHistU); base < nnz; base += waves * (kWave * kHistU)) {
        int32_t c[kHistU];
#pragma unroll
        for (int u = 0; u < kHistU; ++u) {
            const int64_t e = base + u * kWave + lane;
            c[u] = e < nnz ? ci[e] : -1;
        }
#pragma unroll
        for (int u = 0; u < kHistU; ++u) add_bucket_runs(cnt, c[u] >= 0 ? bucket(c[u]) : -1, 1);
    }
    // less the diagonal entries
    for (int64_t r0 = wid * kWave; r0 < m; r0 += waves * kWave) {
        const int64_t r = r0 + lane;
        int b = -1;
        if (r < m) {
            const int64_t a = rp[r], z = rp[r + 1];
            if (z > a && int64_t(ci[z - 1]) == r) b = bucket(r);
        }
        add_bucket_runs(cnt, b, -1);
    }
    __syncthreads();
    for (int x = threadIdx.x; x < nb; x += kBlock)
        if (cnt[x]) atomicAdd(&hist[x], (unsigned long long)(long long)cnt[x]);
}

// column runs of a sorted slab: first[k] / end[k] = first / one-past-last
// record of slab column k (both zero for a column without records).  Four
// records per thread (one 16-byte load), the neighbouring threads' keys by
// shuffles, a load at each wavefront's edges.
constexpr uint32_t kNoKey = 0xffffffffu;  // (slab keys are below 2^31)
__global__ __launch_bounds__(kBlock) void slab_col_runs(const uint32_t* __restrict__ skey, int64_t nrec,
                                                        uint32_t* __restrict__ first, uint32_t* __restrict__ end) {
    const int64_t t = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    const int64_t s0 = 4 * t;
    const int lane = lane_id();
    uint32_t k[4];
    if (s0 + 4 <= nrec && (reinterpret_cast<uintptr_t>(skey) & 15) == 0) {
        const uint4 v = reinterpret_cast<const uint4*>(skey)[t];
        k[0] = v.x;
        k[1] = v.y;
        k[2] = v.z;
        k[3] = v.w;
    } else {
#pragma unroll
        for (int u = 0; u < 4; ++u) k[u] = s0 + u < nrec ? skey[s0 + u] : kNoKey;
    }
    uint32_t prev = __shfl_up(k[3], 1, kWave);
    uint32_t next = __shfl_down(k[0], 1, kWave);
    if (lane == 0) prev = (s0 > 0 && s0 <= nrec) ? skey[s0 - 1] : kNoKey;
    if (lane == kWave - 1) next = s0 + 4 < nrec ? skey[s0 + 4] : kNoKey;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int64_t sx = s0 + u;
        if (sx < nrec) {
            const uint32_t kp = u == 0 ? prev : k[u - 1];
            const uint32_t kn = u == 3 ? next : k[u + 1];
            if (sx == 0 || kp != k[u]) first[k[u]] = uint32_t(sx);
            if (sx == nrec - 1 || kn != k[u]) end[k[u]] = uint32_t(sx + 1);
        }
    }
}

// full row lengths of the slab's columns (lower length + strict-lower
// count), and a zero after them so that the scan also gives the next start
__global__ __launch_bounds__(kBlock) void slab_full_len(const int64_t* __restrict__ rp, int64_t c0, int64_t w,
                                                        const uint32_t* __restrict__ first,
                                                        const uint32_t* __restrict__ end, int64_t* __restrict__ fl) {
    const int64_t k = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (k > w) return;
    fl[k] = k == w ? 0 : (rp[c0 + k + 1] - rp[c0 + k]) + int64_t(end[k] - first[k]);
}

// start of the slab's first full row: the lower entries of the rows before
// c0 (rp[c0]) and the strict-lower entries of the columns before c0
__global__ __launch_bounds__(kBlock) void add_carry(int64_t* __restrict__ a, int64_t w,
                                                    const int64_t* __restrict__ rp_c0, int64_t strict_before) {
    const int64_t k = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (k < w) a[k] += *rp_c0 + strict_before;
}

inline unsigned blocks_for(int64_t n, int64_t per) { return unsigned((n + per - 1) / per); }

}  // namespace

size_t mirror_tile_bytes(int64_t positions) { return size_t((positions + kTileE - 1) / kTileE + 1) * sizeof(int64_t); }

void mirror_tile_rows(const int64_t* rp, int64_t m, int64_t* trow, hipStream_t s) {
    tile_first_rows(rp, m, kTileE, trow, s);
}

void mirror_copy_lower(const MirrorArgs& a, int64_t ebeg, int64_t eend, const int64_t* trow, const int64_t* f_rp,
                       int32_t* f_ci, void* f_val, hipStream_t s) {
    if (eend <= ebeg) return;
    const unsigned nb = blocks_for(eend - ebeg, kTileE);
    if (ebeg != 0) trow = nullptr;  // (the table's tiles start at entry 0)
    if (a.vbytes == 8 && a.val)
        copy_lower<8><<<nb, kBlock, 0, s>>>(a.rp, a.ci, a.val, a.m, ebeg, eend, trow, f_rp, f_ci, f_val);
    else if (a.vbytes == 4 && a.val)
        copy_lower<4><<<nb, kBlock, 0, s>>>(a.rp, a.ci, a.val, a.m, ebeg, eend, trow, f_rp, f_ci, f_val);
    else
        copy_lower<0><<<nb, kBlock, 0, s>>>(a.rp, a.ci, a.val, a.m, ebeg, eend, trow, f_rp, f_ci, f_val);
}

void mirror_coarse_hist(const MirrorArgs& a, int64_t clo, int cb, int nb, unsigned long long* hist,
                        hipStream_t s) {
    (void)hipMemsetAsync(hist, 0, size_t(nb) * sizeof(unsigned long long), s);
    if (a.nnz <= 0 || a.m <= 0) return;
    int64_t grid = (a.nnz + kTileC - 1) / kTileC;
    if (grid > 2048) grid = 2048;
    coarse_hist<<<unsigned(grid), kBlock, 0, s>>>(a.rp, a.ci, a.m, a.nnz, clo, cb, nb, hist);
}

void mirror_slab_columns(const MirrorArgs& a, int64_t c0, int64_t c1, const uint32_t* skey, int64_t nrec,
                         uint32_t* first, uint32_t* end, int64_t* fl, int64_t strict_before, int64_t* f_rp,
                         void* scan_tmp, hipStream_t s) {
    const int64_t w = c1 - c0;
    (void)hipMemsetAsync(first, 0, size_t(w) * sizeof(uint32_t), s);
    (void)hipMemsetAsync(end, 0, size_t(w) * sizeof(uint32_t), s);
    if (nrec > 0) slab_col_runs<<<blocks_for((nrec + 3) / 4, kBlock), kBlock, 0, s>>>(skey, nrec, first, end);
    slab_full_len<<<blocks_for(w + 1, kBlock), kBlock, 0, s>>>(a.rp, c0, w, first, end, fl);
    scan_i64(fl, f_rp + c0, w + 1, nullptr, scan_tmp, s);
    add_carry<<<blocks_for(w + 1, kBlock), kBlock, 0, s>>>(f_rp + c0, w + 1, a.rp + c0, strict_before);
}

void mirror_slab_offsets(int64_t* row_lo, const int64_t* rec_rp, int64_t m, hipStream_t s) {
    if (m > 0) slab_offsets<<<blocks_for(m, kBlock), kBlock, 0, s>>>(row_lo, rec_rp, m);
}

void mirror_slab_counts(const MirrorArgs& a, int64_t c0, int64_t c1, int64_t* row_cnt, int64_t* row_lo,
                        hipStream_t s) {
    if (a.m <= 0) return;
    slab_counts<<<blocks_for(a.m, kBlock), kBlock, 0, s>>>(a.rp, a.ci, a.m, c0, c1, row_cnt, row_lo);
}

void mirror_slab_extract(const MirrorArgs& a, int64_t c0, int64_t nrec, const int64_t* rec_rp, const int64_t* row_lo,
                         int64_t* trow, uint32_t* rkey, uint32_t* rrow, void* rval, hipStream_t s) {
    if (nrec <= 0) return;
    const unsigned nb = blocks_for(nrec, kTileE);
    tile_first_rows(rec_rp, a.m, kTileE, trow, s);
    if (a.vbytes == 8 && a.val)
        slab_extract<8><<<nb, kBlock, 0, s>>>(a.ci, a.val, a.m, c0, nrec, rec_rp, row_lo, trow, rkey, rrow, rval);
    else if (a.vbytes == 4 && a.val)
        slab_extract<4><<<nb, kBlock, 0, s>>>(a.ci, a.val, a.m, c0, nrec, rec_rp, row_lo, trow, rkey, rrow, rval);
    else
        slab_extract<0><<<nb, kBlock, 0, s>>>(a.ci, a.val, a.m, c0, nrec, rec_rp, row_lo, trow, rkey, rrow, rval);
}

void mirror_slab_place(const MirrorArgs& a, int64_t c0, int64_t nrec, const uint32_t* skey, const uint32_t* srow,
                       const void* sval, const uint32_t* first, const int64_t* f_rp, int32_t* f_ci, void* f_val,
                       hipStream_t s) {
    if (nrec <= 0) return;
    const unsigned nb = blocks_for(nrec, kBlock);
    if (a.vbytes == 8 && a.val)
        slab_place<8><<<nb, kBlock, 0, s>>>(a.rp, c0, nrec, skey, srow, sval, first, f_rp, f_ci, f_val);
    else if (a.vbytes == 4 && a.val)
        slab_place<4><<<nb, kBlock, 0, s>>>(a.rp, c0, nrec, skey, srow, sval, first, f_rp, f_ci, f_val);
    else
        slab_place<0><<<nb, kBlock, 0, s>>>(a.rp, c0, nrec, skey, srow, sval, first, f_rp, f_ci, f_val);
}

}  // namespace spsyrk
