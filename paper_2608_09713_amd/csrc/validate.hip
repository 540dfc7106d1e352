// Canonical-CSR checks.
//
// One kernel checks both arrays: workgroup b checks the row pointers of rows
// [b*kTileR, (b+1)*kTileR) and the column ids of entry tile t(b) (tiles of
// kTileE, the radix passes' tiles, dealt to the XCDs in consecutive runs as
// the passes deal them), whose digits it can count for the first radix pass.  Every thread walks a contiguous stretch of entries row by
// row, starting from the row of its first entry (searched in an LDS window of
// the row pointers).  The rows of the workgroup's first entry and of its end
// come from a table written by the rows themselves; a row with out-of-range
// pointers writes nothing, and a missing or inconsistent entry falls back to
// a search.  On a malformed row_ptr every access still stays in bounds (the
// results are then meaningless, but the row check has raised its flag).
#include "common.h"
#include "internal.h"

namespace spsyrk {
namespace {

constexpr int kTileR = 4096;  // row pointers per workgroup
constexpr int kTileE = kRadixTile;  // entries per workgroup
constexpr int kWinV = 2048;   // rows held in LDS
constexpr int kPerE = kTileE / kBlock;

__device__ inline int64_t find_row(const int64_t* rp, int64_t lo, int64_t hi, int64_t e) {
    // largest i in [lo, hi] with rp[i] <= e (for a non-decreasing rp)
    while (lo < hi) {
        const int64_t mid = (lo + hi + 1) >> 1;
        if (rp[mid] <= e)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

// trow[t] = the row holding entry t * kTileE (trow starts at -1).  Rows whose
// pointers lie outside [0, nnz] or decrease write nothing, and a row writes
// at most kRowTiles entries (so a malformed row_ptr costs bounded work; the
// tiles a longer row would cover search for their row instead).
constexpr int64_t kRowTiles = 64;
__global__ __launch_bounds__(kBlock) void entry_tile_rows(const int64_t* __restrict__ rp, int64_t m, int64_t nnz,
                                                          int64_t ntiles, int64_t* __restrict__ trow) {
    const int64_t r = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (r >= m) return;
    const int64_t a = rp[r], b = rp[r + 1];
    if (a < 0 || b < a || b > nnz) return;
    const int64_t t0 = (a + kTileE - 1) / kTileE;
    for (int64_t t = t0; t < ntiles && t * kTileE < b && t < t0 + kRowTiles; ++t) trow[t] = r;
}

__global__ __launch_bounds__(kBlock) void check_csr(const int64_t* __restrict__ rp, const int32_t* __restrict__ ci,
                                                    int64_t m, int64_t n, int64_t nnz, bool upper_forbidden,
                                                    const int64_t* __restrict__ trow, uint32_t* err, FirstHist fh) {
    __shared__ int64_t win[kWinV + 1];
    __shared__ int64_t bounds[2];
    __shared__ uint32_t bad_s;
    __shared__ uint32_t cnt[kWavesPerBlock][256];  // (digit counts, with fh.hist)
    if (threadIdx.x == 0) bad_s = 0;
    if (fh.hist)
        for (int q = 0; q < kWavesPerBlock; ++q) cnt[q][threadIdx.x] = 0;
    __syncthreads();  // (a workgroup with no entries meets no other barrier before its atomics)
    // the entry tile: consecutive tiles on one XCD (workgroups go round-robin
    // over the XCDs), as the radix passes place them
    const int64_t ntiles_e = (nnz + kTileE - 1) / kTileE;
    const int64_t per = (ntiles_e + kXcds - 1) / kXcds;
    // (workgroups past the placed tiles, there for the row pointers only, take none)
    const int64_t etile = int64_t(blockIdx.x) < per * kXcds ? int64_t(blockIdx.x % kXcds) * per + blockIdx.x / kXcds
                                                              : ntiles_e;
    uint32_t bad = 0;
    // row pointers: rp[0] == 0, non-decreasing, inside [0, nnz], rp[m] == nnz
    for (int64_t i = int64_t(blockIdx.x) * kTileR + threadIdx.x;
         i <= m && i < int64_t(blockIdx.x + 1) * kTileR; i += kBlock) {
        const int64_t a = rp[i];
        if (a < 0 || a > nnz || (i == 0 && a != 0) || (i == m && a != nnz)) bad |= kErrRowPtr;
        if (i < m && rp[i + 1] < a) bad |= kErrRowPtr;
    }
    const int64_t e0 = etile * kTileE;
    const int64_t e1 = min(nnz, e0 + kTileE);
    if (etile < ntiles_e) {
        if (threadIdx.x == 0) {
            // row of e0, and a row at or past the row of e1 - 1 (the row of e1)
            int64_t lo = trow[etile];
            if (lo < 0 || lo >= m) lo = find_row(rp, 0, m, e0);
            int64_t hi = e1 < nnz ? trow[etile + 1] : -1;
            if (hi < lo || hi >= m) hi = find_row(rp, 0, m, e1 - 1);
            bounds[0] = lo;
            bounds[1] = hi;
        }
        __syncthreads();
        const int64_t rlo = bounds[0], rhi = bounds[1];
        // (rhi < m always holds for a valid row_ptr; the window reads rp[rhi + 1])
        const bool staged = rhi >= rlo && rhi < m && rhi - rlo + 2 <= kWinV + 1;
        if (staged)
            for (int64_t k = threadIdx.x; k < rhi - rlo + 2; k += kBlock) win[k] = rp[rlo + k];
        __syncthreads();
        // every thread walks kPerE contiguous entries, row by row
        const int64_t ea = e0 + int64_t(threadIdx.x) * kPerE;
        const int64_t eb = min(e1, ea + kPerE);
        if (ea < eb) {
            int64_t r = staged ? rlo + find_row(win, 0, rhi - rlo, ea) : find_row(rp, 0, m, ea);
            int64_t rend = r < m ? (staged ? win[r - rlo + 1] : rp[r + 1]) : nnz;
            int32_t prev = ea > 0 ? ci[ea - 1] : -1;
            bool first = staged ? win[r - rlo] == ea : rp[r] == ea;
            // the stretch's column ids, by 16-byte loads when whole and aligned
            int32_t cc[kPerE];
            if (eb - ea == kPerE && (reinterpret_cast<uintptr_t>(ci + ea) & 15) == 0) {
                const int4* v4 = reinterpret_cast<const int4*>(ci + ea);
#pragma unroll
                for (int u = 0; u < kPerE / 4; ++u) {
                    const int4 q = v4[u];
                    cc[4 * u] = q.x;
                    cc[4 * u + 1] = q.y;
                    cc[4 * u + 2] = q.z;
                    cc[4 * u + 3] = q.w;
                }
            } else {
#pragma unroll
                for (int u = 0; u < kPerE; ++u) cc[u] = ea + u < eb ? ci[ea + u] : 0;
            }
#pragma unroll
            for (int u = 0; u < kPerE; ++u) {
                const int64_t e = ea + u;
                if (e >= eb) break;
                const int32_t c = cc[u];
                if (e >= rend) {
                    // next non-empty row (a malformed row_ptr ends the walk at row m)
                    while (e >= rend && r < m) {
                        ++r;
                        rend = r < m ? (staged && r <= rhi ? win[r - rlo + 1] : rp[r + 1]) : nnz;
                    }
                    first = true;
                }
                if (c < 0 || int64_t(c) >= n) bad |= kErrColRange;
                if (!first && prev >= c) bad |= kErrColOrder;
                if (upper_forbidden && int64_t(c) > r) bad |= kErrUpper;
                prev = c;
                first = false;
            }
            if (fh.hist) {
#pragma unroll
                for (int u = 0; u < kPerE; ++u)
                    if (ea + u < eb) atomicAdd(&cnt[threadIdx.x / kWave][(uint32_t(cc[u]) >> fh.shift) & fh.mask], 1u);
            }
        }
        if (fh.hist) {
            __syncthreads();
            uint32_t t = 0;
#pragma unroll
            for (int q = 0; q < kWavesPerBlock; ++q) t += cnt[q][threadIdx.x];
            fh.hist[int64_t(threadIdx.x) * fh.ntiles + etile] = t;
        }
    }
    if (bad) atomicOr(&bad_s, bad);
    __syncthreads();
    if (threadIdx.x == 0 && bad_s) atomicOr(err, bad_s);
}

__global__ void fill_u32_kernel(uint32_t* p, int64_t n, uint32_t v) {
    int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    for (; i < n; i += stride) p[i] = v;
}

}  // namespace

void fill_u32(uint32_t* p, int64_t n, uint32_t v, hipStream_t s) {
    if (n <= 0) return;
    int64_t blocks = (n + kBlock - 1) / kBlock;
    if (blocks > 65536) blocks = 65536;
    fill_u32_kernel<<<dim3(unsigned(blocks)), dim3(kBlock), 0, s>>>(p, n, v);
}

size_t validate_tmp_bytes(int64_t nnz) { return size_t((nnz + kTileE - 1) / kTileE + 1) * sizeof(int64_t); }

void validate_csr(const DevCsr& A, bool upper_forbidden, uint32_t* err, void* tmp, hipStream_t s,
                  const FirstHist* fh) {
    const int64_t rb = (A.m + 1 + kTileR - 1) / kTileR;
    const int64_t eb = (A.nnz + kTileE - 1) / kTileE;
    const int64_t ebx = (eb + kXcds - 1) / kXcds * kXcds;  // every entry tile placed (see check_csr)
    const int64_t nb = rb > ebx ? rb : ebx;
    const FirstHist h = fh && eb > 0 ? *fh : FirstHist();
    int64_t* trow = static_cast<int64_t*>(tmp);
    if (eb > 0) {
        fill_u32(reinterpret_cast<uint32_t*>(trow), 2 * eb, 0xffffffffu, s);
        if (A.m > 0)
            entry_tile_rows<<<unsigned((A.m + kBlock - 1) / kBlock), kBlock, 0, s>>>(A.rp, A.m, A.nnz, eb, trow);
    }
    check_csr<<<dim3(unsigned(nb)), dim3(kBlock), 0, s>>>(A.rp, A.ci, A.m, A.n, A.nnz, upper_forbidden, trow, err, h);
}

}  // namespace spsyrk
