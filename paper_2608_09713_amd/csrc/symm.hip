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
#include "common.h"
#include "internal.h"

namespace spsyrk {
namespace {

constexpr int kTileS = 2048;              // entries per workgroup
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

}  // namespace

size_t symm_tmp_bytes(int64_t m, int64_t k, int64_t nnz) {
    const size_t wb = (size_t(m) * size_t(k) * sizeof(double) + 255) & ~size_t(255);
    return wb + size_t((nnz + kTileS - 1) / kTileS + 1) * sizeof(int64_t);
}

void symm_product(const DevCsr& C, int sr, const void* x, int64_t ldx, int64_t k, void* y, int64_t ldy, void* tmp,
                  hipStream_t s) {
    double* w = static_cast<double*>(tmp);
    const size_t wb = (size_t(C.m) * size_t(k) * sizeof(double) + 255) & ~size_t(255);
    int64_t* trow = reinterpret_cast<int64_t*>(static_cast<char*>(tmp) + wb);
    zero_f64<<<grid_for(C.m * k), kBlock, 0, s>>>(w, C.m * k);
    if (C.nnz > 0) {
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
