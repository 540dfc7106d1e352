// Partner runs of all entries, and the compaction of staged light rows.
//
// The runs kernel is the memory-latency-bound half of the light path: one
// thread per entry, no LDS beyond a window of row pointers, so many
// wavefronts keep their directory and key loads in flight together.  Its
// output (two words per entry) is read back in entry order by the light-row
// kernel.
#include "common.h"
#include "internal.h"
#include "lookup.h"

namespace spsyrk {
namespace {

constexpr int kTileE = 2048;
constexpr int kWin = 2048;

__device__ inline int64_t last_leq(const int64_t* a, int64_t lo, int64_t hi, int64_t x) {
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

template <bool LOWER>
__global__ __launch_bounds__(kBlock) void runs_kernel(const int64_t* __restrict__ rp, const int32_t* __restrict__ ci,
                                                      int64_t m, int64_t nnz, const uint32_t* __restrict__ key,
                                                      const uint32_t* __restrict__ gptr, int gs, int rowbits,
                                                      const unsigned long long* __restrict__ prod,
                                                      uint32_t* __restrict__ run_lo, uint32_t* __restrict__ run_hi) {
    __shared__ int64_t win[kWin + 1];
    __shared__ int64_t bounds[2];
    const int64_t e0 = int64_t(blockIdx.x) * kTileE;
    const int64_t e1 = min(nnz, e0 + kTileE);
    if (threadIdx.x == 0) {
        bounds[0] = last_leq(rp, 0, m, e0);
        bounds[1] = last_leq(rp, 0, m, e1 - 1);
    }
    __syncthreads();
    const int64_t rlo = bounds[0], rhi = bounds[1];
    const bool staged = rhi - rlo + 2 <= kWin + 1;
    if (staged)
        for (int64_t k = threadIdx.x; k < rhi - rlo + 2; k += kBlock) win[k] = rp[rlo + k];
    __syncthreads();
    constexpr int kPer = kTileE / kBlock;
    uint32_t kk[kPer];
    int64_t row[kPer];
    bool need[kPer];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
        const int64_t e = e0 + u * kBlock + threadIdx.x;
        need[u] = e < e1;
        kk[u] = need[u] ? uint32_t(ci[e]) : 0u;
        int64_t r = 0;
        if (need[u]) r = staged ? rlo + last_leq(win, 0, rhi - rlo, e) : last_leq(rp, rlo, rhi, e);
        row[u] = r;
    }
    if (prod) {
#pragma unroll
        for (int u = 0; u < kPer; ++u)
            if (need[u] && prod[row[u]] == 0) {
                need[u] = false;
                const int64_t e = e0 + u * kBlock + threadIdx.x;
                run_lo[e] = 0;
                run_hi[e] = 0;
            }
    }
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
        if (!need[u]) continue;
        const int64_t e = e0 + u * kBlock + threadIdx.x;
        uint32_t st, len;
        partner_run(key, gptr, gs, rowbits, kk[u], uint32_t(row[u]), LOWER, st, len);
        run_lo[e] = st;
        run_hi[e] = st + len;
    }
}

template <int VB>
__global__ __launch_bounds__(kBlock) void compact_kernel(int64_t m, int64_t staged, const int64_t* __restrict__ ubp,
                                                         const int64_t* __restrict__ row_cnt,
                                                         const int64_t* __restrict__ c_rp,
                                                         const int32_t* __restrict__ s_ci, const void* __restrict__ s_val,
                                                         int32_t* __restrict__ c_ci, void* __restrict__ c_val) {
    __shared__ int64_t win[kWin + 1];
    __shared__ int64_t bounds[2];
    const int64_t s0 = int64_t(blockIdx.x) * kTileE;
    const int64_t s1 = min(staged, s0 + kTileE);
    if (threadIdx.x == 0) {
        bounds[0] = last_leq(ubp, 0, m, s0);
        bounds[1] = last_leq(ubp, 0, m, s1 - 1);
    }
    __syncthreads();
    const int64_t rlo = bounds[0], rhi = bounds[1];
    const bool win_ok = rhi - rlo + 2 <= kWin + 1;
    if (win_ok)
        for (int64_t k = threadIdx.x; k < rhi - rlo + 2; k += kBlock) win[k] = ubp[rlo + k];
    __syncthreads();
    for (int64_t sl = s0 + threadIdx.x; sl < s1; sl += kBlock) {
        const int64_t i = win_ok ? rlo + last_leq(win, 0, rhi - rlo, sl) : last_leq(ubp, rlo, rhi, sl);
        const int64_t off = sl - ubp[i];
        if (off >= row_cnt[i]) continue;
        const int64_t p = c_rp[i] + off;
        c_ci[p] = s_ci[sl];
        if constexpr (VB == 8) static_cast<uint64_t*>(c_val)[p] = static_cast<const uint64_t*>(s_val)[sl];
        if constexpr (VB == 4) static_cast<uint32_t*>(c_val)[p] = static_cast<const uint32_t*>(s_val)[sl];
    }
}

}  // namespace

void partner_runs(const DevCsr& A, const ColIndex& cx, bool lower, const unsigned long long* prod, uint32_t* run_lo,
                  uint32_t* run_hi, hipStream_t s) {
    if (A.nnz <= 0) return;
    const unsigned nb = unsigned((A.nnz + kTileE - 1) / kTileE);
    if (lower)
        runs_kernel<true><<<nb, kBlock, 0, s>>>(A.rp, A.ci, A.m, A.nnz, cx.key, cx.gptr, cx.gs, cx.rowbits, prod,
                                                run_lo, run_hi);
    else
        runs_kernel<false><<<nb, kBlock, 0, s>>>(A.rp, A.ci, A.m, A.nnz, cx.key, cx.gptr, cx.gs, cx.rowbits, prod,
                                                 run_lo, run_hi);
}

void compact_rows(int64_t m, int64_t staged, const int64_t* ubp, const int64_t* row_cnt, const int64_t* c_rp,
                  const int32_t* s_ci, const void* s_val, int vbytes, int32_t* c_ci, void* c_val, hipStream_t s) {
    if (staged <= 0 || m <= 0) return;
    const unsigned nb = unsigned((staged + kTileE - 1) / kTileE);
    if (vbytes == 8)
        compact_kernel<8><<<nb, kBlock, 0, s>>>(m, staged, ubp, row_cnt, c_rp, s_ci, s_val, c_ci, c_val);
    else if (vbytes == 4)
        compact_kernel<4><<<nb, kBlock, 0, s>>>(m, staged, ubp, row_cnt, c_rp, s_ci, s_val, c_ci, c_val);
    else
        compact_kernel<0><<<nb, kBlock, 0, s>>>(m, staged, ubp, row_cnt, c_rp, s_ci, s_val, c_ci, c_val);
}

}  // namespace spsyrk
