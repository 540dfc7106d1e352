// Gustavson accumulation for rows with many products (rows of power-law
// graphs that meet hub columns): one workgroup per row, taken from a work
// queue.
//
// The row's output column range is swept in windows of kWin columns.  In a
// window the row's distinct columns are first marked in an LDS bitmap; a scan
// of the words' popcounts gives every marked column its rank, i.e. its
// position among the row's output entries, so the window's column indices are
// written straight from the bitmap, in order.  The values are then summed in
// LDS over the compacted ranks (tiles of kAcc ranks), so the accumulator only
// spans columns that occur.  Every partner run is sorted by row, so each run
// is consumed front to back through a per-entry cursor: a short stretch of a
// run by a group of kGrp lanes, a long one by a whole wavefront, both over
// contiguous keys.
//
// The symbolic pass builds the bitmaps only and counts the row's columns; the
// numeric pass rebuilds them, writes the column indices and the values.
#include "common.h"
#include "internal.h"
#include "lookup.h"

namespace spsyrk {
namespace {

constexpr int kHB = 512;                 // threads per workgroup
constexpr int kHW = kHB / kWave;         // wavefronts per workgroup
constexpr int kChunkE = 512;             // entries examined per activity round
constexpr int kLongU = 2;                // keys per lane per step of a long walk
constexpr int kHeavyGroups = 1024;       // workgroups of a heavy-row launch
constexpr int kGrp = 8;                  // lanes per short stretch of a walk

// Output columns per window and ranks per value tile: the symbolic pass
// holds a 32 KiB bitmap; the numeric pass a 16 KiB bitmap, the rank of every
// 128 columns' first column (4 KiB) and a 28 KiB value tile, about 52 KiB
// with the activity lists, so that three workgroups share a compute unit
// (windows of 2^17 columns measure 2% faster than 2^16 with a rank per word;
// with twice the LDS only two workgroups fit, and rows wait longer on their
// walks' latency).
template <int SR, bool NUM>
struct HeavyCfg {
    using Acc = typename SrTraits<SR>::Acc;
    static constexpr int kWin = NUM ? (1 << 17) : (1 << 18);
    static constexpr int kWords = kWin / 32;
    static constexpr int kAcc = 28672 / int(sizeof(Acc));
};

// exclusive scan over the kHB threads of a workgroup; *total gets the sum
__device__ inline uint32_t scan_hb(uint32_t v, uint32_t* wt, uint32_t* total) {
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    const uint32_t inc = wave_inclusive_scan(v);
    if (lane == kWave - 1) wt[w] = inc;
    __syncthreads();
    uint32_t off = 0, tot = 0;
#pragma unroll
    for (int q = 0; q < kHW; ++q) {
        const uint32_t t = wt[q];
        if (q < w) off += t;
        tot += t;
    }
    __syncthreads();
    *total = tot;
    return off + inc - v;
}

// Three workgroups of the numeric pass share a compute unit by their LDS;
// that takes six wavefronts per SIMD, i.e. at most 80 VGPRs (with 88, only two
// workgroups fit and the pass takes about 40% longer).
template <int SR, bool NUM, bool LOWER>
__global__ __launch_bounds__(kHB) __attribute__((amdgpu_waves_per_eu(NUM ? 6 : 8)))
void heavy_kernel(HeavyArgs a, int* queue) {
    using Tr = SrTraits<SR>;
    using In = typename Tr::In;
    using Acc = typename Tr::Acc;
    using Out = typename Tr::Out;
    constexpr int kAcc = HeavyCfg<SR, NUM>::kAcc;
    constexpr int kWin = HeavyCfg<SR, NUM>::kWin;
    constexpr int kWords = HeavyCfg<SR, NUM>::kWords;
    constexpr bool kVal = (SR == kF64 || SR == kF32);

    __shared__ __align__(16) uint32_t bits[kWords];
    __shared__ uint32_t prefw[NUM ? kWords / 4 : 1];  // rank of the first column of each 4 words in the window
    __shared__ Acc acc[NUM ? kAcc : 1];
    __shared__ int32_t act_short[kChunkE];
    __shared__ int32_t act_long[kChunkE];
    __shared__ int nshort_s, nlong_s;
    __shared__ int row_s;
    __shared__ uint32_t wt[kHW];
    __shared__ double wtd[kHW];

    const int tid = threadIdx.x;
    const int w = tid / kWave;
    const int lane = lane_id();
    const uint32_t* __restrict__ key = a.cx.key;
    const uint32_t rowmask = a.cx.rowbits >= 32 ? 0xffffffffu : ((1u << a.cx.rowbits) - 1u);
    const int nheavy = *a.heavy_count;

    // rank of column j of the current window among the window's columns
    auto rank_of = [&](int64_t B0, uint32_t j) -> uint32_t {
        if constexpr (!NUM) return 0u;  // (ranks exist in the numeric pass only)
        const uint32_t x = uint32_t(int64_t(j) - B0);
        const uint4 q = reinterpret_cast<const uint4*>(bits)[x >> 7];
        const uint32_t wd[4] = {q.x, q.y, q.z, q.w};
        const uint32_t k = (x >> 5) & 3u, mk = (1u << (x & 31)) - 1u;
        uint32_t r = prefw[x >> 7];
#pragma unroll
        for (uint32_t i = 0; i < 4; ++i) r += i < k ? uint32_t(__popc(wd[i])) : (i == k ? uint32_t(__popc(wd[i] & mk)) : 0u);
        return r;
    };

    // Walk the partner runs of entries [c0, c1) from their cursors through
    // the partners below column B1 (and, for values, of rank below T0 + tl):
    // mark them in the bitmap, or add their terms to the value tile.  Short
    // stretches (under a wavefront of partners) are walked by groups of kGrp
    // lanes, long ones by whole wavefronts.  The cursors move if advance is set.
    // Called by all threads.
    auto walk = [&](int64_t c0, int64_t c1, int64_t B0, int64_t B1, bool value, uint32_t T0, uint32_t tl,
                    bool advance) {
        if (tid == 0) {
            nshort_s = 0;
            nlong_s = 0;
        }
        __syncthreads();
        const uint32_t rlim = T0 + tl;
        for (int64_t e = c0 + tid; e < c1; e += kHB) {
            const uint32_t c = a.cursor[e];
            const uint32_t hi = a.rend[e];
            if (c >= hi) continue;
            const uint32_t j = key[c] & rowmask;
            if (int64_t(j) >= B1 || (value && rank_of(B0, j) >= rlim)) continue;
            bool lng = c + uint32_t(kWave) <= hi;
            if (lng) {
                const uint32_t jl = key[c + kWave - 1] & rowmask;
                lng = int64_t(jl) < B1 && !(value && rank_of(B0, jl) >= rlim);
            }
            if (lng)
                act_long[atomicAdd(&nlong_s, 1)] = int32_t(e - c0);
            else
                act_short[atomicAdd(&nshort_s, 1)] = int32_t(e - c0);
        }
        __syncthreads();
        const int nshort = nshort_s, nlong = nlong_s;
        // short stretches: a group of kGrp lanes each, kGrp consecutive keys
        // per step (the keys in range form a prefix of the stretch)
        {
            const int gl = lane % kGrp;
            for (int q = tid / kGrp; q < nshort; q += kHB / kGrp) {
                const int64_t e = c0 + act_short[q];
                uint32_t c = a.cursor[e];
                const uint32_t hi = a.rend[e];
                double av = 0.0;
                if constexpr (kVal) av = value ? double(static_cast<const In*>(a.val)[e]) : 0.0;
                while (c < hi) {
                    const uint32_t p = c + uint32_t(gl);
                    const uint32_t jj = p < hi ? (key[p] & rowmask) : 0xffffffffu;
                    bool in = false;
                    if (int64_t(jj) < B1) {
                        const uint32_t x = uint32_t(int64_t(jj) - B0);
                        if (value) {
                            const uint32_t rk = rank_of(B0, jj);
                            in = rk >= T0 && rk < rlim;
                            if (in) {
                                if constexpr (NUM) {
                                    if constexpr (kVal)
                                        atomicAdd(&acc[rk - T0], av * double(static_cast<const In*>(a.cx.val)[p]));
                                    else
                                        atomicAdd(&acc[rk - T0], 1);
                                }
                            }
                        } else {
                            in = true;
                            atomicOr(&bits[x >> 5], 1u << (x & 31));
                        }
                    }
                    const uint64_t bal = __ballot(in);
                    const uint32_t took = uint32_t(__popcll((bal >> (lane - gl)) & ((uint64_t(1) << kGrp) - 1)));
                    c += took;
                    if (took < uint32_t(kGrp)) break;
                }
                if (advance && gl == 0) a.cursor[e] = c;
            }
        }
        // long stretches: a wavefront each, kLongU keys per lane per step
        for (int q = w; q < nlong; q += kHW) {
            const int64_t e = c0 + act_long[q];
            uint32_t c = a.cursor[e];
            const uint32_t hi = a.rend[e];
            double av = 0.0;
            if constexpr (kVal) av = value ? double(static_cast<const In*>(a.val)[e]) : 0.0;
            while (c < hi) {
                uint32_t jj[kLongU];
#pragma unroll
                for (int u = 0; u < kLongU; ++u) {
                    const uint32_t p = c + uint32_t(u * kWave) + lane;
                    jj[u] = p < hi ? (key[p] & rowmask) : 0xffffffffu;
                }
                uint32_t took = 0;
                bool full = true;
#pragma unroll
                for (int u = 0; u < kLongU; ++u) {
                    const uint32_t p = c + uint32_t(u * kWave) + lane;
                    bool in = false;
                    if (full && int64_t(jj[u]) < B1) {
                        const uint32_t x = uint32_t(int64_t(jj[u]) - B0);
                        if (value) {
                            const uint32_t rk = rank_of(B0, jj[u]);
                            in = rk >= T0 && rk < rlim;
                            if (in) {
                                if constexpr (NUM) {
                                    if constexpr (kVal)
                                        atomicAdd(&acc[rk - T0], av * double(static_cast<const In*>(a.cx.val)[p]));
                                    else
                                        atomicAdd(&acc[rk - T0], 1);
                                }
                            }
                        } else {
                            in = true;
                            atomicOr(&bits[x >> 5], 1u << (x & 31));
                        }
                    }
                    const uint32_t t = uint32_t(__popcll(__ballot(in)));
                    took += t;
                    full = full && t == uint32_t(kWave);
                }
                c += took;
                if (!full) break;
            }
            if (advance && lane == 0) a.cursor[e] = c;
        }
        __syncthreads();
    };

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
        for (int64_t e = e0 + tid; e < e1; e += kHB) {
            uint2 rr;
            if (!NUM && !a.runs_ready) {
                uint32_t st, len;
                partner_run(key, a.cx.gptr, a.cx.gs, a.cx.rowbits, uint32_t(a.ci[e]), uint32_t(i), LOWER, st, len);
                rr = make_uint2(st, st + len);
                a.run.r8[e] = rr;
                prod_local += len;
            } else {
                rr = run_of(a.run, e);
            }
            a.cursor[e] = rr.x;
            a.rend[e] = rr.y;
        }
        if constexpr (!NUM) {
            const uint64_t tot = wave_reduce_sum(prod_local);
            if (lane == 0 && tot && a.products) atomicAdd(a.products, (unsigned long long)tot);
        }
        __threadfence_block();
        __syncthreads();

        const int64_t jmax = LOWER ? int64_t(i) : a.m_right;
        int64_t count = 0;                          // symbolic: distinct columns so far
        int64_t outp = NUM ? a.c_rp[i] : 0;         // numeric: first output slot of the window
        for (int64_t B0 = 0; B0 < jmax; B0 += kWin) {
            const int64_t B1 = min(jmax, B0 + int64_t(kWin));
            const int nw = int((B1 - B0 + 31) >> 5);
            for (int x = tid; x < nw; x += kHB) bits[x] = 0;
            __syncthreads();

            // mark the window's columns; the numeric pass walks the runs again
            // for the values, so only the symbolic pass moves the cursors here
            for (int64_t c0 = e0; c0 < e1; c0 += kChunkE)
                walk(c0, min(e1, c0 + int64_t(kChunkE)), B0, B1, false, 0u, 0u, !NUM);

            // ranks: every thread owns a contiguous stretch of words
            constexpr int kPer = (kWords + kHB - 1) / kHB;
            const int wlo = min(nw, tid * kPer), whi = min(nw, wlo + kPer);
            uint32_t s = 0;
            for (int x = wlo; x < whi; ++x) s += uint32_t(__popc(bits[x]));
            uint32_t Nw;
            uint32_t off = scan_hb(s, wt, &Nw);
            if constexpr (!NUM) {
                count += Nw;
                __syncthreads();
            } else {
                for (int x = wlo; x < whi; ++x) {
                    if ((x & 3) == 0) prefw[x >> 2] = off;
                    uint32_t b = bits[x];
                    // the window's column indices, in order
                    while (b) {
                        const int t = __ffs(b) - 1;
                        b &= b - 1;
                        SPSYRK_CHECK(outp + off < a.c_rp[i + 1], kDbgHeavyOut);
                        a.c_ci[outp + off] = int32_t(B0 + 32 * x + t);
                        ++off;
                    }
                }
                // (the barrier orders these writes for the workgroup's reads below)
                __syncthreads();

                // values over the compacted ranks, kAcc ranks at a time; an
                // entry joins a value tile only if its next partner's rank
                // falls inside it
                for (uint32_t T0 = 0; T0 < Nw; T0 += uint32_t(kAcc)) {
                    const uint32_t tl = min(Nw - T0, uint32_t(kAcc));
                    for (uint32_t x = tid; x < tl; x += kHB) acc[x] = Acc(0);
                    __syncthreads();
                    for (int64_t c0 = e0; c0 < e1; c0 += kChunkE)
                        walk(c0, min(e1, c0 + int64_t(kChunkE)), B0, B1, true, T0, tl, true);
                    for (uint32_t x = tid; x < tl; x += kHB) {
                        const int64_t p = outp + T0 + x;
                        SPSYRK_CHECK(p < a.c_rp[i + 1], kDbgHeavyOut);
                        Out ov;
                        if constexpr (kVal) {
                            ov = Out(acc[x]);
                        } else if constexpr (SR == kCount) {
                            ov = acc[x];
                        } else {
                            const int32_t j = a.c_ci[p];
                            ov = jaccard(acc[x], E, a.rp_right[j + 1] - a.rp_right[j]);
                        }
                        static_cast<Out*>(a.c_val)[p] = ov;
                    }
                    __syncthreads();
                }
                outp += Nw;
            }
        }
        if constexpr (NUM) {
            if (tid == 0) SPSYRK_CHECK(outp + (LOWER ? 1 : 0) == a.c_rp[i + 1], kDbgHeavyCount);
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
                for (int64_t e = e0 + tid; e < e1; e += kHB) {
                    const double v = double(static_cast<const In*>(a.val)[e]);
                    s += v * v;
                }
                s = wave_reduce_sum(s);
                if (lane == 0) wtd[w] = s;
                __syncthreads();
                double t = 0.0;
                for (int q = 0; q < kHW; ++q) t += wtd[q];
                dv = Out(t);
                __syncthreads();
            } else if constexpr (SR == kCount) {
                dv = int32_t(E);
            } else {
                dv = jaccard(int32_t(E), E, E);
            }
            if (tid == 0) {
                SPSYRK_CHECK(outp < a.c_rp[i + 1], kDbgHeavyOut);
                a.c_ci[outp] = i;
                static_cast<Out*>(a.c_val)[outp] = dv;
            }
        }
        __syncthreads();
    }
}

template <int SR, bool NUM>
void launch(const HeavyArgs& a, int* queue, hipStream_t s) {
    if (a.heavy_max <= 0) return;
    (void)hipMemsetAsync(queue, 0, sizeof(int), s);
    const int64_t grid = a.heavy_max < kHeavyGroups ? a.heavy_max : kHeavyGroups;

    if (a.lower)
        heavy_kernel<SR, NUM, true><<<unsigned(grid), kHB, 0, s>>>(a, queue);
    else
        heavy_kernel<SR, NUM, false><<<unsigned(grid), kHB, 0, s>>>(a, queue);
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
