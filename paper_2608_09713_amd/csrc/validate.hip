// Canonical-CSR checks and the entry -> row map.
#include "common.h"
#include "internal.h"

namespace spsyrk {
namespace {

// row_ptr[0] == 0, non-decreasing, row_ptr[m] == nnz; marks row starts.
__global__ __launch_bounds__(kBlock) void check_rows(const int64_t* __restrict__ rp, int64_t m, int64_t nnz,
                                                     uint32_t* __restrict__ start_bits, uint32_t* err) {
    const int64_t i = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (i > m) return;
    const int64_t a = rp[i];
    if (i == 0 && a != 0) atomicOr(err, kErrRowPtr);
    if (i == m) {
        if (a != nnz) atomicOr(err, kErrRowPtr);
        return;
    }
    const int64_t b = rp[i + 1];
    if (b < a || a < 0 || b > nnz) {
        atomicOr(err, kErrRowPtr);
        return;
    }
    if (b > a) atomicOr(&start_bits[a >> 5], 1u << (a & 31));
}

// column range, strict increase inside rows, optional col <= row
__global__ __launch_bounds__(kBlock) void check_cols(const int64_t* __restrict__ rp, const int32_t* __restrict__ ci,
                                                     int64_t m, int64_t n, int64_t nnz,
                                                     const uint32_t* __restrict__ start_bits, bool upper_forbidden,
                                                     uint32_t* err) {
    const int64_t e = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (e >= nnz) return;
    const int32_t c = ci[e];
    uint32_t bad = 0;
    if (c < 0 || int64_t(c) >= n) bad |= kErrColRange;
    const bool is_start = (start_bits[e >> 5] >> (e & 31)) & 1u;
    if (e > 0 && !is_start && ci[e - 1] >= c) bad |= kErrColOrder;
    if (upper_forbidden) {
        // row of e: last i with rp[i] <= e (only needed for this check)
        int64_t lo = 0, hi = m;
        while (lo < hi) {
            int64_t mid = (lo + hi + 1) >> 1;
            if (rp[mid] <= e)
                lo = mid;
            else
                hi = mid - 1;
        }
        if (int64_t(c) > lo) bad |= kErrUpper;
    }
    if (bad) atomicOr(err, bad);
}

// rows[e] for the entries of one tile of kTileE entries; the tile's row_ptr
// window is staged in LDS when it fits, otherwise rows are searched in place.
constexpr int kTileE = 4096;
constexpr int kRowWin = 4096;

__device__ inline int64_t find_row(const int64_t* rp, int64_t lo, int64_t hi, int64_t e) {
    // largest i in [lo, hi] with rp[i] <= e
    while (lo < hi) {
        int64_t mid = (lo + hi + 1) >> 1;
        if (rp[mid] <= e)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

__global__ __launch_bounds__(kBlock) void rows_of_entries(const int64_t* __restrict__ rp, int64_t m, int64_t nnz,
                                                          uint32_t* __restrict__ rows) {
    __shared__ int64_t win[kRowWin + 1];
    __shared__ int64_t r_lo_s, r_hi_s;
    const int64_t e0 = int64_t(blockIdx.x) * kTileE;
    const int64_t e1 = min(nnz, e0 + kTileE);
    if (threadIdx.x == 0) {
        r_lo_s = find_row(rp, 0, m, e0);
        r_hi_s = find_row(rp, 0, m, e1 - 1);
    }
    __syncthreads();
    const int64_t r_lo = r_lo_s, r_hi = r_hi_s;
    const int64_t nwin = r_hi - r_lo + 2;  // rp[r_lo .. r_hi + 1]
    if (nwin <= kRowWin + 1) {
        for (int64_t k = threadIdx.x; k < nwin; k += kBlock) win[k] = rp[r_lo + k];
        __syncthreads();
        for (int64_t e = e0 + threadIdx.x; e < e1; e += kBlock) {
            int lo = 0, hi = int(nwin - 2);
            while (lo < hi) {
                int mid = (lo + hi + 1) >> 1;
                if (win[mid] <= e)
                    lo = mid;
                else
                    hi = mid - 1;
            }
            rows[e] = uint32_t(r_lo + lo);
        }
    } else {
        for (int64_t e = e0 + threadIdx.x; e < e1; e += kBlock) rows[e] = uint32_t(find_row(rp, r_lo, r_hi, e));
    }
}

__global__ void fill_u32_kernel(uint32_t* p, int64_t n, uint32_t v) {
    int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    for (; i < n; i += stride) p[i] = v;
}

}  // namespace

size_t validate_tmp_bytes(const DevCsr& A) { return size_t((A.nnz + 31) / 32 + 1) * sizeof(uint32_t); }

void fill_u32(uint32_t* p, int64_t n, uint32_t v, hipStream_t s) {
    if (n <= 0) return;
    int64_t blocks = (n + kBlock - 1) / kBlock;
    if (blocks > 65536) blocks = 65536;
    fill_u32_kernel<<<dim3(unsigned(blocks)), dim3(kBlock), 0, s>>>(p, n, v);
}

void validate_csr(const DevCsr& A, bool upper_forbidden, uint32_t* start_bits, uint32_t* err, hipStream_t s) {
    fill_u32(start_bits, (A.nnz + 31) / 32 + 1, 0u, s);
    const int64_t nb_rows = (A.m + 1 + kBlock - 1) / kBlock;
    check_rows<<<dim3(unsigned(nb_rows)), dim3(kBlock), 0, s>>>(A.rp, A.m, A.nnz, start_bits, err);
    if (A.nnz > 0) {
        const int64_t nb = (A.nnz + kBlock - 1) / kBlock;
        check_cols<<<dim3(unsigned(nb)), dim3(kBlock), 0, s>>>(A.rp, A.ci, A.m, A.n, A.nnz, start_bits,
                                                              upper_forbidden, err);
    }
}

void entry_rows(const DevCsr& A, uint32_t* rows, hipStream_t s) {
    if (A.nnz <= 0) return;
    const int64_t nb = (A.nnz + kTileE - 1) / kTileE;
    rows_of_entries<<<dim3(unsigned(nb)), dim3(kBlock), 0, s>>>(A.rp, A.m, A.nnz, rows);
}

}  // namespace spsyrk
