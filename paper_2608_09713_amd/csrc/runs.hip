// Per-row product counts from the partner runs, the compaction of the staged
// light rows into the final CSR arrays, the row of every tile start, and the
// partner runs of an off-diagonal block from dense column starts.
#include "common.h"
#include "internal.h"
#include "lookup.h"

namespace spsyrk {
namespace {

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

// prod[i] = sum of the run lengths of row i's entries.  Every thread walks a
// contiguous stretch of kPerT entries of the workgroup's tile, adding up the
// lengths row by row.  A row that lies inside the stretch is stored at once;
// the partial sums of rows cut by a stretch's ends meet in LDS, and a row cut
// by the tile's ends is added atomically (prod starts at zero).
constexpr int kPerT = 12;
constexpr int kTileP = kBlock * kPerT;
static_assert(kTileP == kRadixTile, "the row products take the validation's tile table");
constexpr int kWinP = 1024;

// trow[t] = the row holding position t * T, for every tile start t * T <
// rp[m] (each such position lies in exactly one non-empty row, which writes it)
__global__ __launch_bounds__(kBlock) void tile_rows(const int64_t* __restrict__ rp, int64_t m, int64_t T,
                                                    int64_t* __restrict__ trow) {
    const int64_t r = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (r >= m) return;
    const int64_t a = rp[r], b = rp[r + 1];
    for (int64_t t = (a + T - 1) / T; t * T < b; ++t) trow[t] = r;
}

__global__ __launch_bounds__(kBlock) void rowprod_kernel(const int64_t* __restrict__ rp, int64_t m, int64_t nnz,
                                                         const RunTab run,
                                                         const int64_t* __restrict__ trow,
                                                         unsigned long long* __restrict__ prod) {
    __shared__ int64_t win[kWinP + 1];
    __shared__ unsigned long long part[kWinP];
    __shared__ uint32_t cut[kWinP];
    __shared__ int64_t bounds[2];
    const int64_t e0 = int64_t(blockIdx.x) * kTileP;
    const int64_t e1 = min(nnz, e0 + kTileP);
    const int64_t a = e0 + int64_t(threadIdx.x) * kPerT;
    const int64_t b = min(e1, a + kPerT);
    // the stretch's run words, loaded first so that they arrive while the
    // tile's rows are set up (16-byte loads for a whole aligned stretch)
    uint32_t w[kPerT];
    if (b - a == kPerT && (reinterpret_cast<uintptr_t>(run.r4 + a) & 15) == 0) {
        const uint4* v4 = reinterpret_cast<const uint4*>(run.r4 + a);
#pragma unroll
        for (int u = 0; u < kPerT / 4; ++u) {
            const uint4 q = nt_load4(v4 + u);
            w[4 * u] = q.x;
            w[4 * u + 1] = q.y;
            w[4 * u + 2] = q.z;
            w[4 * u + 3] = q.w;
        }
    } else {
#pragma unroll
        for (int u = 0; u < kPerT; ++u) w[u] = a + u < b ? run.r4[a + u] : 0u;
    }
    if (threadIdx.x == 0) {
        // rows of the tile's first entry and (at most one row past the tile)
        // of its end, from the tile table; the last tile searches for its
        // end, and so does a tile the table leaves out (-1)
        int64_t lo = trow[blockIdx.x];
        if (lo < 0) lo = last_leq(rp, 0, m, e0);
        int64_t hi = e1 < nnz ? trow[blockIdx.x + 1] : -1;
        if (hi < 0) hi = last_leq(rp, lo, m, e1 < nnz ? e1 : e1 - 1);
        bounds[0] = lo;
        bounds[1] = hi;
    }
    __syncthreads();
    const int64_t rlo = bounds[0], rhi = bounds[1];
    const int64_t nrw = rhi - rlo + 1;
    const bool staged = nrw <= kWinP;
    if (staged)
        for (int64_t k = threadIdx.x; k <= nrw; k += kBlock) {
            win[k] = rp[rlo + k];
            if (k < nrw) {
                part[k] = 0;
                cut[k] = 0;
            }
        }
    __syncthreads();
    if (a < b) {
        uint32_t rl[kPerT];
#pragma unroll
        for (int u = 0; u < kPerT; ++u) {
            const uint2 r = a + u < b ? run_from(run, w[u], a + u) : make_uint2(0u, 0u);
            rl[u] = r.y - r.x;
        }
        // row of the stretch's first entry and its bounds
        int64_t r = staged ? rlo + last_leq(win, 0, rhi - rlo, a) : last_leq(rp, rlo, rhi, a);
        int64_t rstart = staged ? win[r - rlo] : rp[r];
        int64_t rend = staged ? win[r - rlo + 1] : rp[r + 1];
        unsigned long long acc = 0;
        for (int u = 0; u < kPerT; ++u) {
            const int64_t e = a + u;
            if (e >= b) break;
            if (e >= rend) {
                // the finished row ends inside the stretch
                if (rstart >= a) {
                    prod[r] = acc;
                } else if (staged) {
                    atomicAdd(&part[r - rlo], acc);
                    cut[r - rlo] = 1;
                } else if (acc) {
                    atomicAdd(&prod[r], acc);
                }
                acc = 0;
                do {  // the row of e (empty rows keep their zero)
                    ++r;
                    rstart = rend;
                    rend = staged ? win[r - rlo + 1] : rp[r + 1];
                } while (rend <= e);
            }
            acc += rl[u];
        }
        if (rstart >= a && rend <= b) {
            prod[r] = acc;
        } else if (staged) {
            atomicAdd(&part[r - rlo], acc);
            cut[r - rlo] = 1;
        } else if (acc) {
            atomicAdd(&prod[r], acc);
        }
    }
    __syncthreads();
    if (staged)
        for (int64_t k = threadIdx.x; k < nrw; k += kBlock) {
            if (!cut[k]) continue;
            if (win[k] >= e0 && win[k + 1] <= e1)
                prod[rlo + k] = part[k];
            else if (part[k])
                atomicAdd(&prod[rlo + k], part[k]);
        }
}

constexpr int kCTile = 4096;  // staging slots per compaction workgroup
constexpr int kCTileSmall = 512;  // the same for few slots (compact_tile)
template <int VB>
struct SlotT {  // a staged value of VB bytes (a placeholder for VB 0)
    using T = uint32_t;
};
template <>
struct SlotT<8> {
    using T = uint64_t;
};
constexpr int kCWin = 512;    // rows held in LDS by a compaction workgroup

// Staged words of packed count and Jaccard outputs (see FusedArgs::pack_rr):
// the column and the value, from the count, the row's length and (Jaccard)
// the partner's length.  The quotients come from double products (exact for
// words below 2^32 and divisors below 2^17; see run_from).
struct Unpack {
    uint32_t rr = 0, r2 = 0;
    double inv_rr = 0.0, inv_r2 = 0.0;
};
template <int PK>
__device__ inline void unpack_store(const Unpack& u, uint32_t w, int64_t len_i, int64_t p, int32_t* c_ci, void* c_val) {
    const uint32_t j = uint32_t(fma(double(w), u.inv_rr, 0x1p-18));
    const uint32_t rem = w - j * u.rr;
    c_ci[p] = int32_t(j);
    if constexpr (PK == 1) {
        static_cast<int32_t*>(c_val)[p] = int32_t(rem);
    } else {
        const uint32_t cnt = uint32_t(fma(double(rem), u.inv_r2, 0x1p-18));
        const uint32_t lenj = rem - cnt * u.r2;
        static_cast<float*>(c_val)[p] = jaccard(int32_t(cnt), len_i, int64_t(lenj));
    }
}

// PK 0: columns and VB-byte values copied; PK 1 (counts) and 2 (Jaccard):
// packed words unpacked (rp_a: the row pointers of A, for the row lengths)
template <int VB, int PK, int CT>
__global__ __launch_bounds__(kBlock) void compact_kernel(int64_t m, int64_t staged, const int64_t* __restrict__ ubp,
                                                         const int64_t* __restrict__ trow,
                                                         const int64_t* __restrict__ row_cnt,
                                                         const int64_t* __restrict__ c_rp,
                                                         const int32_t* __restrict__ s_ci, const void* __restrict__ s_val,
                                                         int32_t* __restrict__ c_ci, void* __restrict__ c_val,
                                                         const int64_t* __restrict__ rp_a, Unpack un) {
    __shared__ int64_t wub[kCWin + 1];  // staging slot of the window's rows
    __shared__ int64_t wend[kCWin];     // end of each row's valid staged entries
    __shared__ int64_t wdel[kCWin];     // final position minus staging slot
    __shared__ int32_t wlen[PK == 2 ? kCWin : 1];  // (Jaccard) the rows' lengths
    __shared__ uint16_t rowof[CT];  // window row of every slot of the tile
    __shared__ uint32_t wt[kWavesPerBlock];
    __shared__ int64_t bounds[2];
    const int64_t s0 = int64_t(blockIdx.x) * CT;
    const int64_t s1 = min(staged, s0 + CT);
    // a whole tile's staged columns (or packed words) are loaded first, so
    // that they arrive while the tile's rows are set up
    constexpr int kPerC = CT / kBlock;
    const bool whole = s1 - s0 == CT;
    int32_t pre[kPerC];
    if (whole)
#pragma unroll
        for (int i = 0; i < kPerC; ++i) pre[i] = s_ci[s0 + i * kBlock + threadIdx.x];
    if (threadIdx.x == 0) {
        // rows of the tile's first slot and (at most one row past the tile)
        // of its end, from the tile table; the last tile searches for its end
        const int64_t lo = trow[blockIdx.x];
        bounds[0] = lo;
        bounds[1] = s1 < staged ? trow[blockIdx.x + 1] : last_leq(ubp, lo, m, s1 - 1);
    }
    __syncthreads();
    const int64_t rlo = bounds[0], rhi = bounds[1];
    const int64_t nrw = rhi - rlo + 1;
    const bool win_ok = nrw <= kCWin;
    if (win_ok) {
        for (int x = threadIdx.x; x < CT; x += kBlock) rowof[x] = 0;
        for (int64_t k = threadIdx.x; k <= nrw; k += kBlock) {
            const int64_t u = ubp[rlo + k];
            wub[k] = u;
            if (k == nrw) break;
            wend[k] = u + row_cnt[rlo + k];
            wdel[k] = c_rp[rlo + k] - u;
            if constexpr (PK == 2) wlen[k] = int32_t(rp_a[rlo + k + 1] - rp_a[rlo + k]);
        }
        __syncthreads();
        // every row with staging room in the tile marks its first slot (a row
        // without room shares its slot with a later row and marks nothing),
        // then a max-scan gives each slot its row
        for (int64_t k = 1 + threadIdx.x; k < nrw; k += kBlock)
            if (wub[k] < wub[k + 1] && wub[k] < s1) rowof[wub[k] - s0] = uint16_t(k);
        __syncthreads();
        constexpr int kPer = CT / kBlock;
        const int lane = lane_id();
        const int w = threadIdx.x / kWave;
        uint32_t run_max = 0;
#pragma unroll
        for (int q = 0; q < kPer; ++q) run_max = max(run_max, uint32_t(rowof[threadIdx.x * kPer + q]));
        uint32_t inc = run_max;
#pragma unroll
        for (int d = 1; d < kWave; d <<= 1) {
            const uint32_t u = __shfl_up(inc, d, kWave);
            if (lane >= d) inc = max(inc, u);
        }
        if (lane == kWave - 1) wt[w] = inc;
        __syncthreads();
        uint32_t before = 0;
        for (int q = 0; q < w; ++q) before = max(before, wt[q]);
        const uint32_t prev = __shfl_up(inc, 1, kWave);
        if (lane > 0) before = max(before, prev);
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            before = max(before, uint32_t(rowof[threadIdx.x * kPer + q]));
            rowof[threadIdx.x * kPer + q] = uint16_t(before);
        }
    }
    __syncthreads();
    if (win_ok && whole) {
        // a whole tile: the slots of a thread in batches of kBatch, every
        // batch's loads in flight together before its stores
        using V = typename SlotT<VB>::T;
        constexpr int kBatch = CT / kBlock < 8 ? CT / kBlock : 8;
        static_assert(CT % (kBlock * kBatch) == 0, "whole batches per tile");
#pragma unroll
        for (int b = 0; b < CT / (kBlock * kBatch); ++b) {
            int32_t cv[kBatch];
            V vv[kBatch];
            bool live[kBatch];
#pragma unroll
            for (int q = 0; q < kBatch; ++q) {
                const int x = (b * kBatch + q) * kBlock + threadIdx.x;
                live[q] = s0 + x < wend[rowof[x]];
                cv[q] = pre[b * kBatch + q];
                if (live[q]) {
                    if constexpr (VB != 0) vv[q] = static_cast<const V*>(s_val)[s0 + x];
                }
            }
#pragma unroll
            for (int q = 0; q < kBatch; ++q) {
                const int x = (b * kBatch + q) * kBlock + threadIdx.x;
                if (live[q]) {
                    const int64_t p = s0 + x + wdel[rowof[x]];
                    SPSYRK_CHECK(p >= 0 && p < c_rp[m], kDbgCompactOut);
                    if constexpr (PK != 0) {
                        unpack_store<PK>(un, uint32_t(cv[q]), PK == 2 ? int64_t(wlen[rowof[x]]) : 0, p, c_ci, c_val);
                    } else {
                        c_ci[p] = cv[q];
                        if constexpr (VB != 0) static_cast<V*>(c_val)[p] = vv[q];
                    }
                }
            }
        }
        return;
    }
    for (int64_t sl = s0 + threadIdx.x; sl < s1; sl += kBlock) {
        int64_t end, del, len_i = 0;
        if (win_ok) {
            const int k = rowof[sl - s0];
            end = wend[k];
            del = wdel[k];
            if constexpr (PK == 2) len_i = wlen[k];
        } else {
            const int64_t i = last_leq(ubp, rlo, rhi, sl);
            end = ubp[i] + row_cnt[i];
            del = c_rp[i] - ubp[i];
            if constexpr (PK == 2) len_i = rp_a[i + 1] - rp_a[i];
        }
        if (sl >= end) continue;
        const int64_t p = sl + del;
        SPSYRK_CHECK(p >= 0 && p < c_rp[m], kDbgCompactOut);
        if constexpr (PK != 0) {
            unpack_store<PK>(un, uint32_t(s_ci[sl]), len_i, p, c_ci, c_val);
            continue;
        }
        c_ci[p] = s_ci[sl];
        if constexpr (VB == 8) static_cast<uint64_t*>(c_val)[p] = static_cast<const uint64_t*>(s_val)[sl];
        if constexpr (VB == 4) static_cast<uint32_t*>(c_val)[p] = static_cast<const uint32_t*>(s_val)[sl];
    }
}

// entries per column (scanned into column starts by the caller)
__global__ __launch_bounds__(kBlock) void count_columns(const int32_t* __restrict__ ci, int64_t nnz,
                                                        uint32_t* __restrict__ cnt) {
    for (int64_t e = int64_t(blockIdx.x) * kBlock + threadIdx.x; e < nnz; e += int64_t(gridDim.x) * kBlock)
        atomicAdd(&cnt[ci[e]], 1u);
}

// the partners of entry e of the left operand are the whole column ci[e] of
// the right operand
__global__ __launch_bounds__(kBlock) void offdiag_runs_kernel(const int32_t* __restrict__ ci, int64_t nnz,
                                                              const uint32_t* __restrict__ cptr,
                                                              const RunTab run) {
    const int64_t e = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (e >= nnz) return;
    const int32_t c = ci[e];
    set_run(run, e, cptr[c], cptr[c + 1]);
}

// out[k] = rp[r0 + k] - rp[r0] for k in [0, m]: the row pointers of rows
// [r0, r0 + m) of a CSR matrix as a matrix of their own
__global__ __launch_bounds__(kBlock) void rebase_rows_kernel(const int64_t* __restrict__ rp, int64_t r0, int64_t m,
                                                             int64_t* __restrict__ out) {
    const int64_t k = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (k <= m) out[k] = rp[r0 + k] - rp[r0];
}

__global__ __launch_bounds__(kBlock) void shift_columns_kernel(int32_t* __restrict__ ci, int64_t nnz, int32_t off) {
    for (int64_t p = int64_t(blockIdx.x) * kBlock + threadIdx.x; p < nnz; p += int64_t(gridDim.x) * kBlock)
        ci[p] += off;
}

template <typename T>
__global__ __launch_bounds__(kBlock) void gather_kernel(T* __restrict__ dst, const T* __restrict__ src,
                                                        const uint32_t* __restrict__ idx, int64_t n) {
    for (int64_t p = int64_t(blockIdx.x) * kBlock + threadIdx.x; p < n; p += int64_t(gridDim.x) * kBlock)
        dst[p] = src[idx[p]];
}

}  // namespace

void gather_values(void* dst, const void* src, const uint32_t* idx, int64_t n, int vb, hipStream_t s) {
    if (n <= 0) return;
    int64_t blocks = (n + kBlock - 1) / kBlock;
    if (blocks > 65536) blocks = 65536;
    if (vb == 8)
        gather_kernel<uint64_t><<<unsigned(blocks), kBlock, 0, s>>>(static_cast<uint64_t*>(dst),
                                                                     static_cast<const uint64_t*>(src), idx, n);
    else
        gather_kernel<uint32_t><<<unsigned(blocks), kBlock, 0, s>>>(static_cast<uint32_t*>(dst),
                                                                     static_cast<const uint32_t*>(src), idx, n);
}

void rebase_rows(const int64_t* rp, int64_t r0, int64_t m, int64_t* out, hipStream_t s) {
    rebase_rows_kernel<<<unsigned((m + 1 + kBlock - 1) / kBlock), kBlock, 0, s>>>(rp, r0, m, out);
}

void shift_columns(int32_t* ci, int64_t nnz, int32_t off, hipStream_t s) {
    if (nnz <= 0 || off == 0) return;
    int64_t blocks = (nnz + kBlock - 1) / kBlock;
    if (blocks > 65536) blocks = 65536;
    shift_columns_kernel<<<unsigned(blocks), kBlock, 0, s>>>(ci, nnz, off);
}

namespace {
__global__ __launch_bounds__(kBlock) void heavy_sums_kernel(const int32_t* __restrict__ rows, int64_t n,
                                                            const int64_t* __restrict__ rp,
                                                            const int64_t* __restrict__ c_rp,
                                                            unsigned long long* __restrict__ out) {
    unsigned long long e = 0, o = 0;
    for (int64_t q = int64_t(blockIdx.x) * kBlock + threadIdx.x; q < n; q += int64_t(gridDim.x) * kBlock) {
        const int64_t r = rows[q];
        e += (unsigned long long)(rp[r + 1] - rp[r]);
        o += (unsigned long long)(c_rp[r + 1] - c_rp[r]);
    }
    e = wave_reduce_sum(e);
    o = wave_reduce_sum(o);
    if (lane_id() == 0 && (e | o)) {
        atomicAdd(out, e);
        atomicAdd(out + 1, o);
    }
}
}  // namespace

void heavy_sums(const int32_t* rows, int64_t n, const int64_t* rp, const int64_t* c_rp, unsigned long long* out,
                hipStream_t s) {
    if (n <= 0) return;
    int64_t grid = (n + kBlock - 1) / kBlock;
    if (grid > 256) grid = 256;
    heavy_sums_kernel<<<unsigned(grid), kBlock, 0, s>>>(rows, n, rp, c_rp, out);
}

namespace {
// sort key of a heavy row: rows with more products first (63 - bits of the count)
__global__ __launch_bounds__(kBlock) void heavy_order_keys(const int32_t* __restrict__ rows, int64_t n,
                                                           const unsigned long long* __restrict__ prod,
                                                           uint32_t* __restrict__ key) {
    const int64_t q = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (q < n) key[q] = uint32_t(63 - bit_width_u64(prod[rows[q]]));
}
}  // namespace

size_t heavy_order_tmp_bytes(int64_t n) {
    return 3 * ((size_t(n) * sizeof(uint32_t) + 255) & ~size_t(255)) + radix_tmp_bytes(n);
}

void heavy_order(int32_t* rows, int64_t n, const unsigned long long* prod, void* tmp, hipStream_t s) {
    if (n <= 1) return;
    const size_t a = (size_t(n) * sizeof(uint32_t) + 255) & ~size_t(255);
    uint32_t* ka = static_cast<uint32_t*>(tmp);
    uint32_t* kb = reinterpret_cast<uint32_t*>(static_cast<char*>(tmp) + a);
    uint32_t* rb = reinterpret_cast<uint32_t*>(static_cast<char*>(tmp) + 2 * a);
    void* rtmp = static_cast<char*>(tmp) + 3 * a;
    heavy_order_keys<<<unsigned((n + kBlock - 1) / kBlock), kBlock, 0, s>>>(rows, n, prod, ka);
    uint32_t* ra = reinterpret_cast<uint32_t*>(rows);
    if (radix_sort(ka, kb, ra, rb, nullptr, nullptr, 0, n, 6, rtmp, s))
        (void)hipMemcpyAsync(rows, rb, size_t(n) * sizeof(uint32_t), hipMemcpyDeviceToDevice, s);
}

void tile_first_rows(const int64_t* rp, int64_t m, int64_t T, int64_t* trow, hipStream_t s) {
    if (m <= 0) return;
    tile_rows<<<unsigned((m + kBlock - 1) / kBlock), kBlock, 0, s>>>(rp, m, T, trow);
}

void column_starts(const int32_t* ci, int64_t nnz, int64_t n, uint32_t* cptr, void* scan_tmp, hipStream_t s) {
    (void)hipMemsetAsync(cptr, 0, size_t(n + 1) * sizeof(uint32_t), s);
    if (nnz > 0) {
        int64_t grid = (nnz + kBlock - 1) / kBlock;
        if (grid > 65536) grid = 65536;
        count_columns<<<unsigned(grid), kBlock, 0, s>>>(ci, nnz, cptr);
    }
    scan_u32(cptr, cptr, n + 1, nullptr, scan_tmp, s);
}

void offdiag_runs(const int32_t* ci, int64_t nnz, const uint32_t* cptr, const RunTab& run, hipStream_t s) {
    if (nnz <= 0) return;
    offdiag_runs_kernel<<<unsigned((nnz + kBlock - 1) / kBlock), kBlock, 0, s>>>(ci, nnz, cptr, run);
}

size_t row_products_tmp_bytes(int64_t nnz) { return size_t((nnz + kTileP - 1) / kTileP + 1) * sizeof(int64_t); }

void row_products(const int64_t* rp, int64_t m, int64_t nnz, const RunTab& run, void* tmp, unsigned long long* prod,
                  hipStream_t s, const int64_t* trow1) {
    if (nnz <= 0 || m <= 0) return;
    const unsigned nb = unsigned((nnz + kTileP - 1) / kTileP);
    int64_t* trow = static_cast<int64_t*>(tmp);
    if (trow1)
        trow = const_cast<int64_t*>(trow1);
    else
        tile_first_rows(rp, m, kTileP, trow, s);
    rowprod_kernel<<<nb, kBlock, 0, s>>>(rp, m, nnz, run, trow, prod);
}

// Staging slots per compaction workgroup: kCTile, or for fewer slots than
// 256 such tiles (fewer workgroups than compute units) tiles of kCTileSmall,
// so that more workgroups share the work.
static int compact_tile(int64_t staged) { return staged < int64_t(256) * kCTile ? kCTileSmall : kCTile; }

size_t compact_tmp_bytes(int64_t staged) {
    const int ct = compact_tile(staged);
    return size_t((staged + ct - 1) / ct + 1) * sizeof(int64_t);
}

template <int CT>
static void launch_compact(int64_t m, int64_t staged, const int64_t* ubp, const int64_t* row_cnt, const int64_t* c_rp,
                    const int32_t* s_ci, const void* s_val, int vbytes, int64_t* trow, int32_t* c_ci, void* c_val,
                    hipStream_t s, int packed, const Unpack& un, const int64_t* rp_a) {
    const unsigned nb = unsigned((staged + CT - 1) / CT);
    tile_first_rows(ubp, m, CT, trow, s);
    if (packed == kCount)
        compact_kernel<0, 1, CT><<<nb, kBlock, 0, s>>>(m, staged, ubp, trow, row_cnt, c_rp, s_ci, s_val, c_ci, c_val,
                                                       rp_a, un);
    else if (packed == kJaccard)
        compact_kernel<0, 2, CT><<<nb, kBlock, 0, s>>>(m, staged, ubp, trow, row_cnt, c_rp, s_ci, s_val, c_ci, c_val,
                                                       rp_a, un);
    else if (vbytes == 8)
        compact_kernel<8, 0, CT><<<nb, kBlock, 0, s>>>(m, staged, ubp, trow, row_cnt, c_rp, s_ci, s_val, c_ci, c_val,
                                                       rp_a, un);
    else if (vbytes == 4)
        compact_kernel<4, 0, CT><<<nb, kBlock, 0, s>>>(m, staged, ubp, trow, row_cnt, c_rp, s_ci, s_val, c_ci, c_val,
                                                       rp_a, un);
    else
        compact_kernel<0, 0, CT><<<nb, kBlock, 0, s>>>(m, staged, ubp, trow, row_cnt, c_rp, s_ci, s_val, c_ci, c_val,
                                                       rp_a, un);
}

void compact_rows(int64_t m, int64_t staged, const int64_t* ubp, const int64_t* row_cnt, const int64_t* c_rp,
                  const int32_t* s_ci, const void* s_val, int vbytes, void* tmp, int32_t* c_ci, void* c_val,
                  hipStream_t s, int packed, uint32_t pack_rr, uint32_t pack_r2, const int64_t* rp_a) {
    if (staged <= 0 || m <= 0) return;
    int64_t* trow = static_cast<int64_t*>(tmp);
    Unpack un;
    if (packed) {
        un.rr = pack_rr;
        un.r2 = pack_r2 ? pack_r2 : 1u;
        un.inv_rr = 1.0 / double(un.rr);
        un.inv_r2 = 1.0 / double(un.r2);
    }
    if (compact_tile(staged) == kCTile)
        launch_compact<kCTile>(m, staged, ubp, row_cnt, c_rp, s_ci, s_val, vbytes, trow, c_ci, c_val, s, packed, un,
                               rp_a);
    else
        launch_compact<kCTileSmall>(m, staged, ubp, row_cnt, c_rp, s_ci, s_val, vbytes, trow, c_ci, c_val, s, packed,
                                    un, rp_a);
}

}  // namespace spsyrk
