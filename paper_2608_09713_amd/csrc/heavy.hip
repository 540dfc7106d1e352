// Gustavson accumulation for rows with many products (hub rows of power-law
// graphs): one workgroup per row, taken from a work queue.  The row's output
// column range is swept in tiles; a tile is a dense accumulator in LDS (a
// value per column plus an occupancy byte), so the tile's output comes out in
// column order with no sort.  Every partner run is sorted by row, so each run
// is consumed front to back through a per-entry cursor: a tile only touches
// the runs whose next element falls inside it, and those are read with whole
// wavefronts over contiguous keys.
//
// The symbolic pass finds the partner runs (kept per entry for the numeric
// pass) and counts distinct columns per tile with occupancy bytes only; the
// numeric pass accumulates values with LDS atomics and writes each tile's
// occupied columns in order.
#include "common.h"
#include "internal.h"
#include "lookup.h"

namespace spsyrk {
namespace {

constexpr int kChunkE = 1024;  // entries scanned per activity round

template <int SR, bool NUM>
struct TileCfg {
    // columns per tile: 32 KiB of occupancy bytes for counting, 32 KiB of
    // accumulators (8 or 4 bytes each) plus their occupancy for values, so
    // that three workgroups share a compute unit
    static constexpr int kW = !NUM ? 32768 : ((SR == kF64 || SR == kF32) ? 4096 : 8192);
};

template <int SR, bool NUM, bool LOWER>
__global__ __launch_bounds__(kBlock) void heavy_kernel(HeavyArgs a, int* queue) {
    using Tr = SrTraits<SR>;
    using In = typename Tr::In;
    using Acc = typename Tr::Acc;
    using Out = typename Tr::Out;
    constexpr int kW = TileCfg<SR, NUM>::kW;
    constexpr bool kVal = (SR == kF64 || SR == kF32);

    __shared__ uint8_t occ[kW];
    __shared__ Acc acc[NUM ? kW : 1];
    __shared__ int32_t act[kChunkE];
    __shared__ int nact_s;
    __shared__ int row_s;
    __shared__ uint32_t wt[kWavesPerBlock];
    __shared__ uint64_t wt64[kWavesPerBlock];
    __shared__ double wtd[kWavesPerBlock];

    const int tid = threadIdx.x;
    const int w = tid / kWave;
    const int lane = lane_id();
    const uint32_t* __restrict__ key = a.cx.key;
    const uint32_t rowmask = a.cx.rowbits >= 32 ? 0xffffffffu : ((1u << a.cx.rowbits) - 1u);
    const int nheavy = *a.heavy_count;

    if constexpr (NUM) {
        for (int x = tid; x < kW; x += kBlock) acc[x] = Acc(0);
    }

    while (true) {
        if (tid == 0) {
            const int h = atomicAdd(queue, 1);
            row_s = h < nheavy ? a.heavy_rows[h] : -1;
        }
        __syncthreads();
        const int i = row_s;
        __syncthreads();
        if (i < 0) break;
        const int64_t e0 = a.rp[i], e1 = a.rp[i + 1];
        const int64_t E = e1 - e0;

        // partner runs and cursors
        uint64_t prod_local = 0;
        for (int64_t e = e0 + tid; e < e1; e += kBlock) {
            uint32_t st, len;
            if (!NUM && !a.runs_ready) {
                partner_run(key, a.cx.gptr, a.cx.gs, a.cx.rowbits, uint32_t(a.ci[e]), uint32_t(i), LOWER, st, len);
                a.run[e] = make_uint2(st, st + len);
                prod_local += len;
            } else {
                st = a.run[e].x;
            }
            a.cursor[e] = st;
        }
        if constexpr (!NUM) {
            uint64_t tot = wave_reduce_sum(prod_local);
            if (lane == 0 && tot && a.products) atomicAdd(a.products, (unsigned long long)tot);
        }
        __threadfence_block();
        __syncthreads();

        const int64_t jmax = LOWER ? int64_t(i) : a.m_right;
        int64_t count = 0;                          // symbolic: distinct columns so far
        int64_t outp = NUM ? a.c_rp[i] : 0;         // numeric: next output slot
        for (int64_t W0 = 0; W0 < jmax; W0 += kW) {
            const int64_t W1 = min(jmax, W0 + int64_t(kW));
            const int span = int(W1 - W0);
            for (int x = tid; x < span; x += kBlock) occ[x] = 0;
            __syncthreads();
            for (int64_t c0 = e0; c0 < e1; c0 += kChunkE) {
                const int64_t c1 = min(e1, c0 + int64_t(kChunkE));
                if (tid == 0) nact_s = 0;
                __syncthreads();
                for (int64_t e = c0 + tid; e < c1; e += kBlock) {
                    const uint32_t c = a.cursor[e];
                    if (c < a.run[e].y && int64_t(key[c] & rowmask) < W1) act[atomicAdd(&nact_s, 1)] = int32_t(e - e0);
                }
                __syncthreads();
                const int nact = nact_s;
                for (int q = w; q < nact; q += kWavesPerBlock) {
                    const int64_t e = e0 + act[q];
                    uint32_t c = a.cursor[e];
                    const uint32_t hi = a.run[e].y;
                    double av = 0.0;
                    if constexpr (kVal && NUM) av = double(static_cast<const In*>(a.val)[e]);
                    while (c < hi) {
                        const uint32_t p = c + lane;
                        bool in = false;
                        uint32_t j = 0;
                        if (p < hi) {
                            j = key[p] & rowmask;
                            in = int64_t(j) < W1;
                        }
                        const uint64_t m = __ballot(in);
                        if (in) {
                            const int x = int(j - W0);
                            occ[x] = 1;
                            if constexpr (NUM) {
                                if constexpr (kVal)
                                    atomicAdd(&acc[x], av * double(static_cast<const In*>(a.cx.val)[p]));
                                else
                                    atomicAdd(&acc[x], 1);
                            }
                        }
                        const uint32_t took = uint32_t(__popcll(m));
                        c += took;
                        if (took < uint32_t(kWave)) break;
                    }
                    if (lane == 0) a.cursor[e] = c;
                }
                __syncthreads();
            }
            // tile result
            if constexpr (!NUM) {
                uint32_t s = 0;
                for (int x = tid; x < span; x += kBlock) s += occ[x];
                uint32_t tot;
                s = wave_reduce_sum(s);
                if (lane == 0) wt[w] = s;
                __syncthreads();
                tot = 0;
                for (int q = 0; q < kWavesPerBlock; ++q) tot += wt[q];
                __syncthreads();
                count += tot;
            } else {
                // each thread owns a contiguous run of columns of the tile
                const int per = (span + kBlock - 1) / kBlock;
                const int lo = min(span, tid * per), hi = min(span, lo + per);
                uint32_t s = 0;
                for (int x = lo; x < hi; ++x) s += occ[x];
                uint32_t tot;
                uint32_t off = block_exclusive_scan(s, wt, &tot);
                int64_t p = outp + off;
                for (int x = lo; x < hi; ++x) {
                    if (!occ[x]) continue;
                    const int32_t j = int32_t(W0 + x);
                    a.c_ci[p] = j;
                    Out ov;
                    if constexpr (kVal) {
                        ov = Out(acc[x]);
                    } else if constexpr (SR == kCount) {
                        ov = acc[x];
                    } else {
                        ov = jaccard(acc[x], E, a.rp_right[j + 1] - a.rp_right[j]);
                    }
                    static_cast<Out*>(a.c_val)[p] = ov;
                    acc[x] = Acc(0);
                    ++p;
                }
                outp += tot;
                __syncthreads();
            }
        }
        // diagonal (lower triangle only; a heavy row is never empty)
        if constexpr (!NUM) {
            if (tid == 0) {
                a.row_nnz[i] = count + (LOWER ? 1 : 0);
                if (a.nnz_total) atomicAdd(a.nnz_total, (unsigned long long)(count + (LOWER ? 1 : 0)));
            }
        } else if (LOWER) {
            Out dv;
            if constexpr (kVal) {
                // fixed-order reduction of the squared entries
                double s = 0.0;
                for (int64_t e = e0 + tid; e < e1; e += kBlock) {
                    const double v = double(static_cast<const In*>(a.val)[e]);
                    s += v * v;
                }
                s = wave_reduce_sum(s);
                if (lane == 0) wtd[w] = s;
                __syncthreads();
                double t = 0.0;
                for (int q = 0; q < kWavesPerBlock; ++q) t += wtd[q];
                dv = Out(t);
                __syncthreads();
            } else if constexpr (SR == kCount) {
                dv = int32_t(E);
            } else {
                dv = jaccard(int32_t(E), E, E);
            }
            if (tid == 0) {
                a.c_ci[outp] = i;
                static_cast<Out*>(a.c_val)[outp] = dv;
            }
        }
        __syncthreads();
    }
    (void)wt64;
}

template <int SR, bool NUM>
void launch(const HeavyArgs& a, int* queue, hipStream_t s) {
    if (a.heavy_max <= 0) return;
    (void)hipMemsetAsync(queue, 0, sizeof(int), s);
    int64_t grid = a.heavy_max < 2048 ? a.heavy_max : 2048;
    if (a.lower)
        heavy_kernel<SR, NUM, true><<<unsigned(grid), kBlock, 0, s>>>(a, queue);
    else
        heavy_kernel<SR, NUM, false><<<unsigned(grid), kBlock, 0, s>>>(a, queue);
}

template <bool NUM>
void dispatch(const HeavyArgs& a, int* queue, hipStream_t s) {
    switch (a.sr) {
        case kF64: launch<kF64, NUM>(a, queue, s); break;
        case kF32: launch<kF32, NUM>(a, queue, s); break;
        case kCount: launch<kCount, NUM>(a, queue, s); break;
        default: launch<kJaccard, NUM>(a, queue, s); break;
    }
}

}  // namespace

void heavy_symbolic(const HeavyArgs& a, int* queue, hipStream_t s) { dispatch<false>(a, queue, s); }
void heavy_numeric(const HeavyArgs& a, int* queue, hipStream_t s) { dispatch<true>(a, queue, s); }

}  // namespace spsyrk
