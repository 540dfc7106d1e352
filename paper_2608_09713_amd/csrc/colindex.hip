// Column index of the right operand from its column-sorted records.
//
// `pack` writes (column-in-group, row) keys, drops the last entry of every
// column when only partners with a smaller row are ever needed, and fills the
// group directory: the first entry of every column that opens a new group
// writes the directory slots of the groups between the previous column's
// group and its own.  In lower mode it also writes every entry's partner run
// (the entries of its column with a smaller row, which open the column) at
// the entry's index, so the rows never search the index.
#include "common.h"
#include "internal.h"

namespace spsyrk {
namespace {

constexpr int kPTile = 2048;  // positions per pack workgroup

// column starts (first entry of a column) in every pack tile
__global__ __launch_bounds__(kBlock) void tile_starts(const uint32_t* __restrict__ scol, int64_t n,
                                                      uint32_t* __restrict__ tcnt) {
    __shared__ uint32_t wt[kWavesPerBlock];
    const int64_t base = int64_t(blockIdx.x) * kPTile;
    const int64_t end = min(n, base + kPTile);
    uint32_t c = 0;
    for (int64_t p = base + threadIdx.x; p < end; p += kBlock) c += (p == 0 || scol[p] != scol[p - 1]) ? 1u : 0u;
    uint32_t tot;
    (void)block_exclusive_scan(c, wt, &tot);
    if (threadIdx.x == 0) tcnt[blockIdx.x] = tot;
}

template <int VB, bool JAC>
__global__ __launch_bounds__(kBlock) void pack(const uint32_t* __restrict__ scol, const uint32_t* __restrict__ srow,
                                               const uint32_t* __restrict__ sent, const void* __restrict__ vals_b,
                                               RunTab run, int64_t n, const uint32_t* __restrict__ tbase,
                                               bool drop_last, int gs, int rowbits, int lenbits, int64_t ngroups,
                                               const int64_t* __restrict__ nkept, const int64_t* __restrict__ rp_b,
                                               uint32_t* __restrict__ key, void* __restrict__ val,
                                               uint32_t* __restrict__ gptr, uint32_t* __restrict__ vsrc) {
    __shared__ int64_t colstart[kPTile];
    __shared__ uint32_t excl[kPTile];  // column starts before each position
    __shared__ int64_t wt[kWavesPerBlock];
    __shared__ uint32_t wt32[kWavesPerBlock];
    __shared__ int64_t carry_s;
    const int64_t base = int64_t(blockIdx.x) * kPTile;
    const int64_t end = min(n, base + kPTile);
    // column start of the tile's first position (its column may begin in an earlier tile)
    if (threadIdx.x == 0 && run) {
        const uint32_t c0 = scol[base];
        int64_t lo = 0, hi = base;
        while (lo < hi) {
            const int64_t mid = (lo + hi) >> 1;
            if (scol[mid] < c0)
                lo = mid + 1;
            else
                hi = mid;
        }
        carry_s = lo;
    }
    {
        // column starts before each position: the tile's base plus a block scan
        constexpr int kPer = kPTile / kBlock;
        uint32_t sc[kPer];
        uint32_t cnt = 0;
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int64_t p = base + int64_t(threadIdx.x) * kPer + k;
            sc[k] = cnt;
            cnt += (p < end && (p == 0 || scol[p] != scol[p - 1])) ? 1u : 0u;
        }
        uint32_t tot;
        const uint32_t pre = block_exclusive_scan(cnt, wt32, &tot) + tbase[blockIdx.x];
#pragma unroll
        for (int k = 0; k < kPer; ++k) excl[threadIdx.x * kPer + k] = pre + sc[k];
        __syncthreads();
    }
    if (run) {
        // inclusive max-scan of "position if it starts a column" over the tile
        constexpr int kPer = kPTile / kBlock;
        int64_t v[kPer];
        int64_t mx = -1;
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int64_t p = base + int64_t(threadIdx.x) * kPer + k;
            int64_t st = -1;
            if (p < end && (p == 0 || scol[p] != scol[p - 1])) st = p;
            mx = st > mx ? st : mx;
            v[k] = mx;
        }
        // exclusive max over the preceding threads
        int64_t inc = mx;
#pragma unroll
        for (int d = 1; d < kWave; d <<= 1) {
            const int64_t u = __shfl_up(inc, d, kWave);
            if (lane_id() >= d) inc = u > inc ? u : inc;
        }
        if (lane_id() == kWave - 1) wt[threadIdx.x / kWave] = inc;
        __syncthreads();
        int64_t before = carry_s;
        const int w = threadIdx.x / kWave;
        for (int q = 0; q < w; ++q) before = wt[q] > before ? wt[q] : before;
        int64_t prev = __shfl_up(inc, 1, kWave);
        if (lane_id() > 0) before = prev > before ? prev : before;
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int64_t cs = v[k] > before ? v[k] : before;
            colstart[threadIdx.x * kPer + k] = cs;
        }
        __syncthreads();
    }
    const uint32_t gmask = (gs >= 32) ? 0xffffffffu : ((1u << gs) - 1u);
    const uint32_t rowmask = rowbits >= 32 ? 0xffffffffu : ((1u << rowbits) - 1u);
    const uint32_t lmax = lenbits > 0 ? (1u << lenbits) - 1u : 0u;
    for (int64_t p = base + threadIdx.x; p < end; p += kBlock) {
        const uint32_t col = scol[p];
        const bool start = p == 0 || scol[p - 1] != col;
        const bool last = p == n - 1 || scol[p + 1] != col;
        const uint32_t field = srow[p];
        const uint32_t row = field & rowmask;
        // kept entries before p: every column entirely before p lost its last entry
        const int64_t cols_before = int64_t(excl[p - base]) + (start ? 1 : 0) - 1;
        if (run) {
            // partners of this entry (j < row): the kept entries that open its column
            const int64_t rank = p - colstart[p - base];
            if (rank > 0) {
                const int64_t first_kept = drop_last ? colstart[p - base] - cols_before : colstart[p - base];
                set_run(run, sent[p], uint32_t(first_kept), uint32_t(first_kept + rank));
            }
        }
        if (start && gptr) {
            // directory slots of the groups opened by this column
            const int64_t q0 = drop_last ? p - cols_before : p;
            const int64_t g = int64_t(col >> gs);
            const int64_t gprev = p == 0 ? -1 : int64_t(scol[p - 1] >> gs);
            for (int64_t x = gprev + 1; x <= g; ++x) gptr[x] = uint32_t(q0);
        }
        if (p == n - 1 && gptr) {
            const uint32_t kept = uint32_t(*nkept);
            for (int64_t x = int64_t(col >> gs) + 1; x <= ngroups; ++x) gptr[x] = kept;
        }
        int64_t q = p;
        if (drop_last) {
            if (last) continue;
            q = p - cols_before;
        }
        if (vsrc) nt_store(sent[p], vsrc + q);
        if constexpr (JAC) {
            if (!val) {
                nt_store(field, key + q);  // (no directory) the row and its saturated length
            } else {
                nt_store(((col & gmask) << rowbits) | row, key + q);
                const uint32_t lf = lenbits > 0 ? field >> rowbits : lmax;
                nt_store(lf < lmax ? int32_t(lf) : int32_t(rp_b[row + 1] - rp_b[row]), static_cast<int32_t*>(val) + q);
            }
        } else {
            nt_store(((col & gmask) << rowbits) | row, key + q);
        }
        if constexpr (JAC) {
        } else if constexpr (VB == 8) {
            nt_store(static_cast<const uint64_t*>(vals_b)[sent[p]], static_cast<uint64_t*>(val) + q);
        } else if constexpr (VB == 4) {
            nt_store(static_cast<const uint32_t*>(vals_b)[sent[p]], static_cast<uint32_t*>(val) + q);
        }
    }
}

__global__ void kept_count(int64_t n, const uint32_t* ncols_distinct, bool drop_last, int64_t* nkept) {
    *nkept = drop_last ? n - int64_t(*ncols_distinct) : n;
}

__global__ __launch_bounds__(kBlock) void empty_directory(int64_t ngroups, uint32_t* __restrict__ gptr) {
    const int64_t g = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (g <= ngroups) gptr[g] = 0;
}

}  // namespace

size_t colindex_tmp_bytes(int64_t n) {
    const int64_t nt = (n + kPTile - 1) / kPTile;
    return ((size_t(nt + 1) * 4 + 255) & ~size_t(255)) + 256 + scan_tmp_bytes(nt + 1);
}

void build_colindex(const uint32_t* scol, const uint32_t* srow, const uint32_t* sent, int64_t n_entries, bool drop_last,
                    int vbytes_in, int sr, const void* vals_b, const int64_t* rp_b, int lenbits, ColIndex& cx, void* tmp,
                    int64_t* d_nkept, const RunTab& run, hipStream_t s, uint32_t* vsrc) {
    const int64_t ntp = (n_entries + kPTile - 1) / kPTile;
    uint32_t* tbase = static_cast<uint32_t*>(tmp);
    char* after = static_cast<char*>(tmp) + ((size_t(ntp + 1) * 4 + 255) & ~size_t(255));
    uint32_t* ncols = reinterpret_cast<uint32_t*>(after);
    void* scan_tmp = after + 256;
    const int64_t n = n_entries;
    if (n == 0) {
        (void)hipMemsetAsync(d_nkept, 0, sizeof(int64_t), s);
        if (cx.gptr) {
            const unsigned ng = unsigned((cx.ngroups + 1 + kBlock - 1) / kBlock);
            empty_directory<<<ng, kBlock, 0, s>>>(cx.ngroups, cx.gptr);
        }
        return;
    }
    const unsigned np = unsigned(ntp);
    tile_starts<<<np, kBlock, 0, s>>>(scol, n, tbase);
    scan_u32(tbase, tbase, ntp, ncols, scan_tmp, s);
    // the number of distinct columns fixes the kept count and the directory's end
    kept_count<<<1, 1, 0, s>>>(n, ncols, drop_last, d_nkept);
#define SPSYRK_PACK(VBv, JACv)                                                                                    \
    pack<VBv, JACv><<<np, kBlock, 0, s>>>(scol, srow, sent, vals_b, run, n, tbase, drop_last, cx.gs, cx.rowbits,  \
                                          lenbits, cx.ngroups, d_nkept, rp_b, cx.key, cx.val, cx.gptr, vsrc)
    if (sr == kJaccard)
        SPSYRK_PACK(0, true);
    else if (vbytes_in == 8)
        SPSYRK_PACK(8, false);
    else if (vbytes_in == 4)
        SPSYRK_PACK(4, false);
    else
        SPSYRK_PACK(0, false);
#undef SPSYRK_PACK
}

}  // namespace spsyrk
