// Column index of the right operand from its column-sorted records: packs
// (column-in-group, row) keys, drops the last entry of every column when only
// partners with a smaller row are ever needed, and builds the group
// directory by binary search over the sorted columns.
#include "common.h"
#include "internal.h"

namespace spsyrk {
namespace {

__global__ __launch_bounds__(kBlock) void start_flags(const uint32_t* __restrict__ scol, int64_t n,
                                                      uint32_t* __restrict__ st) {
    const int64_t p = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (p >= n) return;
    st[p] = (p == 0 || scol[p] != scol[p - 1]) ? 1u : 0u;
}

template <int VB, bool JAC>
__global__ __launch_bounds__(kBlock) void pack(const uint32_t* __restrict__ scol, const uint32_t* __restrict__ srow,
                                               const void* __restrict__ sval, int64_t n,
                                               const uint32_t* __restrict__ excl, bool drop_last, int gs, int rowbits,
                                               const int64_t* __restrict__ rp_b, uint32_t* __restrict__ key,
                                               void* __restrict__ val) {
    const int64_t p = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (p >= n) return;
    const uint32_t col = scol[p];
    const bool start = p == 0 || scol[p - 1] != col;
    const bool last = p == n - 1 || scol[p + 1] != col;
    int64_t q = p;
    if (drop_last) {
        if (last) return;
        const int64_t cidx = int64_t(excl[p]) + (start ? 1 : 0) - 1;  // columns before this one
        q = p - cidx;
    }
    const uint32_t gmask = (gs >= 32) ? 0xffffffffu : ((1u << gs) - 1u);
    const uint32_t row = srow[p];
    key[q] = ((col & gmask) << rowbits) | row;
    if constexpr (JAC) {
        static_cast<int32_t*>(val)[q] = int32_t(rp_b[row + 1] - rp_b[row]);
    } else if constexpr (VB == 8) {
        static_cast<uint64_t*>(val)[q] = static_cast<const uint64_t*>(sval)[p];
    } else if constexpr (VB == 4) {
        static_cast<uint32_t*>(val)[q] = static_cast<const uint32_t*>(sval)[p];
    }
}

__global__ void kept_count(int64_t n, const uint32_t* ncols_distinct, bool drop_last, int64_t* nkept) {
    *nkept = drop_last ? n - int64_t(*ncols_distinct) : n;
}

__global__ __launch_bounds__(kBlock) void directory(const uint32_t* __restrict__ scol, int64_t n,
                                                    const uint32_t* __restrict__ excl, bool drop_last, int gs,
                                                    int64_t ngroups, const int64_t* __restrict__ nkept,
                                                    uint32_t* __restrict__ gptr) {
    const int64_t g = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (g > ngroups) return;
    const uint64_t target = uint64_t(g) << gs;
    int64_t lo = 0, hi = n;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (uint64_t(scol[mid]) < target)
            lo = mid + 1;
        else
            hi = mid;
    }
    int64_t q = lo;
    if (drop_last) q = (lo < n) ? lo - int64_t(excl[lo]) : *nkept;
    gptr[g] = uint32_t(q);
}

}  // namespace

size_t colindex_tmp_bytes(int64_t n) {
    return ((size_t(n) * 4 + 255) & ~size_t(255)) + 256 + scan_tmp_bytes(n);
}

void build_colindex(const uint32_t* scol, const uint32_t* srow, const void* sval, int64_t n_entries, bool drop_last,
                    int vbytes_in, int sr, const int64_t* rp_b, ColIndex& cx, void* tmp, int64_t* d_nkept,
                    hipStream_t s) {
    uint32_t* excl = static_cast<uint32_t*>(tmp);
    char* after = static_cast<char*>(tmp) + ((size_t(n_entries) * 4 + 255) & ~size_t(255));
    uint32_t* ncols = reinterpret_cast<uint32_t*>(after);
    void* scan_tmp = after + 256;
    const int64_t n = n_entries;
    if (n > 0) {
        const unsigned nb = unsigned((n + kBlock - 1) / kBlock);
        start_flags<<<nb, kBlock, 0, s>>>(scol, n, excl);
        scan_u32(excl, excl, n, ncols, scan_tmp, s);
        const bool jac = sr == kJaccard;
        if (jac)
            pack<0, true><<<nb, kBlock, 0, s>>>(scol, srow, sval, n, excl, drop_last, cx.gs, cx.rowbits, rp_b, cx.key,
                                                cx.val);
        else if (vbytes_in == 8)
            pack<8, false><<<nb, kBlock, 0, s>>>(scol, srow, sval, n, excl, drop_last, cx.gs, cx.rowbits, rp_b, cx.key,
                                                 cx.val);
        else if (vbytes_in == 4)
            pack<4, false><<<nb, kBlock, 0, s>>>(scol, srow, sval, n, excl, drop_last, cx.gs, cx.rowbits, rp_b, cx.key,
                                                 cx.val);
        else
            pack<0, false><<<nb, kBlock, 0, s>>>(scol, srow, sval, n, excl, drop_last, cx.gs, cx.rowbits, rp_b, cx.key,
                                                 cx.val);
        kept_count<<<1, 1, 0, s>>>(n, ncols, drop_last, d_nkept);
    } else {
        (void)hipMemsetAsync(d_nkept, 0, sizeof(int64_t), s);
    }
    const unsigned ng = unsigned((cx.ngroups + 1 + kBlock - 1) / kBlock);
    directory<<<ng, kBlock, 0, s>>>(scol, n, excl, drop_last, cx.gs, cx.ngroups, d_nkept, cx.gptr);
}

}  // namespace spsyrk
