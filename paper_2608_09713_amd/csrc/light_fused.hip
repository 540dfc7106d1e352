// Single-pass Gustavson accumulation of the light rows.
//
// Work unit: a chunk of R consecutive rows per wavefront.  Each wavefront
// works alone in its own slice of LDS (no workgroup barriers), in batches of
// consecutive light rows that fit the LDS budget:
//
//   1. partner runs of the batch's entries (found beforehand, read in entry
//      order);
//   2. products flattened over the entries (the owner entry of every product
//      comes from a scatter of run starts and a max-scan), every key loaded
//      in one round;
//   3. ordered buckets per row (bucket order = column order): count, scan,
//      scatter; inside a bucket each product learns whether it is the first of
//      its column (the leader), the leader's rank among the bucket's distinct
//      columns, and its column's value (terms summed in product order);
//   4. the row is written at its staging slot (row upper bound = products +
//      diagonal, known from the column index), its exact length recorded.
//
// A scan of the exact lengths gives the row pointers and a streaming copy
// moves the rows into place, so no row waits for the lengths of earlier
// rows.  Rows with too many entries or products ("heavy") are left to the
// dense-tile kernel.
#include "common.h"
#include "internal.h"
#include "lookup.h"

namespace spsyrk {
namespace {

constexpr int kFE = kFusedEntries;   // entries per batch
constexpr int kFP = kFusedProducts;  // products per batch
constexpr int kFR = kFusedRows;      // rows per chunk (upper limit)
constexpr int kFB = kFP + kFR;       // buckets per batch
constexpr int kWavesF = 2;           // wavefronts per workgroup
constexpr int kMaxBatches = kFR;


__device__ inline void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int SR>
struct ItemOf {
    using T = int32_t;  // unused (count) or |S(j)|, then the Jaccard bits (Jaccard)
};
template <>
struct ItemOf<kF64> {
    using T = double;
};
template <>
struct ItemOf<kF32> {
    using T = double;
};

template <typename Item>
struct WaveLds {
    int64_t rp[kFR + 1];
    int64_t rcnt[kFR];        // output entries per row; later the row's first output slot
    uint16_t rprod[kFR];      // products of light rows (0 for heavy rows)
    uint16_t rnb[kFR + 1];    // buckets of the row in the current batch
    uint16_t rbb[kFR + 1];    // first bucket of the row in the current batch
    uint64_t rscale[kFR];     // bucket of column j: (j * rscale) >> 32 spreads [0, range) evenly
    uint8_t rlight[kFR];
    uint8_t bra[kMaxBatches + 1], brb[kMaxBatches + 1];  // batches [bra, brb) of the chunk
    uint32_t ent_start[kFE];
    uint16_t ent_len[kFE];
    uint16_t ent_poff[kFE + 1];
    uint8_t ent_row[kFE];
    int16_t owner[kFP];
    uint32_t s_j[kFP];
    uint16_t s_t[kFP];
    uint16_t s_rank[kFP];     // 0xffff marks a product that is not its column's leader
    Item s_v[kFP];
    uint32_t hist[kFB + 1];
    uint32_t ucnt[kFB + 1];
};

// exclusive scan in place of a[0..n) by one wavefront (lane = contiguous segment)
template <typename T>
__device__ inline uint32_t wave_scan_lds(T* a, int n) {
    const int lane = lane_id();
    const int per = (n + kWave - 1) / kWave;
    const int lo = min(n, lane * per), hi = min(n, lo + per);
    uint32_t s = 0;
    for (int x = lo; x < hi; ++x) s += uint32_t(a[x]);
    const uint32_t inc = wave_inclusive_scan(s);
    uint32_t off = inc - s;
    const uint32_t tot = __shfl(inc, kWave - 1, kWave);
    for (int x = lo; x < hi; ++x) {
        const uint32_t v = uint32_t(a[x]);
        a[x] = T(off);
        off += v;
    }
    wave_sync();
    return tot;
}

template <int SR, bool LOWER>
struct Chunk {
    using Tr = SrTraits<SR>;
    using In = typename Tr::In;
    using Out = typename Tr::Out;
    using Item = typename ItemOf<SR>::T;
    static constexpr bool kVal = (SR == kF64 || SR == kF32);

    const FusedArgs& a;
    WaveLds<Item>& L;
    int64_t r0 = 0;
    int lane;
    uint32_t rowmask;
    int jbits_right;

    __device__ Chunk(const FusedArgs& a_, WaveLds<Item>& L_) : a(a_), L(L_) {
        lane = lane_id();
        rowmask = a.cx.rowbits >= 32 ? 0xffffffffu : ((1u << a.cx.rowbits) - 1u);
        jbits_right = bit_width_u64(a.m_right > 1 ? uint64_t(a.m_right - 1) : 0);
    }

    // Partner runs, buckets, leaders and per-bucket distinct counts for the
    // light rows [ra, rb).  The batch's products stay in LDS, sorted by
    // (row, bucket).  If add is set, every row's off-diagonal count is added
    // to rcnt.  Returns the number of products.
    __device__ int batch(int ra, int rb, bool add) {
        const int64_t ebase = L.rp[ra];
        const int ne = int(L.rp[rb] - ebase);
        const uint32_t* __restrict__ key = a.cx.key;
        // partner runs of the batch's entries, found beforehand (runs kernel)
        for (int x = lane; x < ne; x += kWave) {
            const int64_t e = ebase + x;
            int lo = ra, hi = rb - 1;  // last row of the batch starting at or before e
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (L.rp[mid] <= e)
                    lo = mid;
                else
                    hi = mid - 1;
            }
            const uint32_t st = a.run_lo[e];
            const uint32_t len = a.run_hi[e] - st;
            L.ent_start[x] = st;
            L.ent_len[x] = uint16_t(len);
            L.ent_row[x] = uint8_t(lo);
            L.ent_poff[x] = uint16_t(len);
        }
        wave_sync();
        const int P = int(wave_scan_lds(L.ent_poff, ne));
        if (lane == 0) L.ent_poff[ne] = uint16_t(P);
        // per-row buckets: one per product (at most one per possible column);
        // bucket of column j = floor(j * nb / range), monotone in j
        const int nrb = rb - ra;
        uint32_t nb = 0;
        if (lane < nrb) {
            const int r = ra + lane;
            const int64_t range = LOWER ? (r0 + r) : a.m_right;
            uint64_t want = L.rprod[r] > 0 ? L.rprod[r] : 1;
            if (range > 0 && uint64_t(range) < want) want = uint64_t(range);
            nb = uint32_t(want);
            L.rnb[r] = uint16_t(nb);
            L.rscale[r] = range > 0 ? (uint64_t(nb) << 32) / uint64_t(range) : 0;
        }
        const uint32_t inc = wave_inclusive_scan(nb);
        if (lane < nrb) L.rbb[ra + lane] = uint16_t(inc - nb);
        const uint32_t B = __shfl(inc, kWave - 1, kWave);
        for (uint32_t b = lane; b <= B; b += kWave) {
            L.hist[b] = 0;
            L.ucnt[b] = 0;
        }
        // owner entry of every product: run starts scattered, then max-scan
        for (int t = lane; t < P; t += kWave) L.owner[t] = -1;
        wave_sync();
        for (int x = lane; x < ne; x += kWave)
            if (L.ent_len[x]) L.owner[L.ent_poff[x]] = int16_t(x);
        wave_sync();
        {
            const int per = (P + kWave - 1) / kWave;
            const int lo = min(P, lane * per), hi = min(P, lo + per);
            int mx = -1;
            for (int x = lo; x < hi; ++x) mx = max(mx, int(L.owner[x]));
            int incm = mx;
#pragma unroll
            for (int d = 1; d < kWave; d <<= 1) {
                const int u = __shfl_up(incm, d, kWave);
                if (lane >= d) incm = max(incm, u);
            }
            int run = __shfl_up(incm, 1, kWave);
            if (lane == 0) run = -1;
            for (int x = lo; x < hi; ++x) {
                run = max(run, int(L.owner[x]));
                L.owner[x] = int16_t(run);
            }
        }
        wave_sync();
        // products: every key (and partner value) of the lane loaded in one round,
        // kept in registers for both passes
        constexpr int kPV = kFP / kWave;
        uint32_t pj[kPV], pb[kPV];
        Item pv[kPV];
#pragma unroll
        for (int v = 0; v < kPV; ++v) {
            const int t = lane + v * kWave;
            pj[v] = 0;
            pb[v] = 0;
            if (t < P) {
                const int x = L.owner[t];
                const uint32_t pos = L.ent_start[x] + uint32_t(t - L.ent_poff[x]);
                pj[v] = key[pos];
                if constexpr (SR == kJaccard) {
                    pv[v] = static_cast<const int32_t*>(a.cx.val)[pos];
                } else if constexpr (kVal) {
                    pv[v] = double(static_cast<const In*>(a.val)[ebase + x]) *
                            double(static_cast<const In*>(a.cx.val)[pos]);
                }
                pb[v] = uint32_t(L.ent_row[x]);
            }
        }
#pragma unroll
        for (int v = 0; v < kPV; ++v) {
            const int t = lane + v * kWave;
            if (t < P) {
                const uint32_t j = pj[v] & rowmask;
                const int r = int(pb[v]);
                pj[v] = j;
                pb[v] = L.rbb[r] + uint32_t((uint64_t(j) * L.rscale[r]) >> 32);
                atomicAdd(&L.hist[pb[v]], 1u);
            }
        }
        wave_sync();
        wave_scan_lds(L.hist, int(B));
        // scatter into buckets; hist[b] ends as the end of bucket b
#pragma unroll
        for (int v = 0; v < kPV; ++v) {
            const int t = lane + v * kWave;
            if (t < P) {
                const uint32_t q = atomicAdd(&L.hist[pb[v]], 1u);
                L.s_j[q] = pj[v];
                L.s_t[q] = uint16_t(t);
                if constexpr (SR == kJaccard || kVal) L.s_v[q] = pv[v];
            }
        }
        wave_sync();
        // leaders: the first product (in product order) of each column
        for (int q = lane; q < P; q += kWave) {
            const uint32_t j = L.s_j[q];
            const uint32_t t = L.s_t[q];
            const int r = L.ent_row[L.owner[t]];
            const uint32_t b = L.rbb[r] + uint32_t((uint64_t(j) * L.rscale[r]) >> 32);
            const uint32_t lo = b ? L.hist[b - 1] : 0u, hi = L.hist[b];
            bool lead = true;
            if (hi - lo > 1)
                for (uint32_t u = lo; u < hi; ++u)
                    if (L.s_j[u] == j && L.s_t[u] < t) lead = false;
            L.s_rank[q] = lead ? 0 : 0xffff;
        }
        wave_sync();
        // rank among the bucket's distinct columns, and the column's value
        for (int q = lane; q < P; q += kWave) {
            if (L.s_rank[q] == 0xffff) continue;
            const uint32_t j = L.s_j[q];
            const uint32_t t = L.s_t[q];
            const int r = L.ent_row[L.owner[t]];
            const uint32_t b = L.rbb[r] + uint32_t((uint64_t(j) * L.rscale[r]) >> 32);
            const uint32_t lo = b ? L.hist[b - 1] : 0u, hi = L.hist[b];
            uint32_t rank = 0, cnt = 1;
            if (hi - lo > 1) {
                cnt = 0;
                for (uint32_t u = lo; u < hi; ++u) {
                    const uint32_t ju = L.s_j[u];
                    rank += (ju < j && L.s_rank[u] != 0xffff) ? 1u : 0u;
                    cnt += ju == j ? 1u : 0u;
                }
            }
            if constexpr (kVal) {
                double sum = L.s_v[q];
                uint32_t last = t;
                for (uint32_t c = 1; c < cnt; ++c) {
                    uint32_t best = 0xffffffffu, bu = q;
                    for (uint32_t u = lo; u < hi; ++u) {
                        const uint32_t tu = L.s_t[u];
                        if (L.s_j[u] == j && tu > last && tu < best) {
                            best = tu;
                            bu = u;
                        }
                    }
                    sum += L.s_v[bu];
                    last = best;
                }
                L.s_v[q] = sum;
            } else if constexpr (SR == kCount) {
                L.s_v[q] = int32_t(cnt);
            } else {
                const int64_t len_i = L.rp[r + 1] - L.rp[r];
                L.s_v[q] = __float_as_int(jaccard(int32_t(cnt), len_i, L.s_v[q]));
            }
            atomicAdd(&L.ucnt[b], 1u);
            L.s_rank[q] = uint16_t(rank);
        }
        wave_sync();
        const uint32_t U = wave_scan_lds(L.ucnt, int(B));
        if (lane == 0) L.ucnt[B] = U;
        wave_sync();
        if (add && lane < nrb) {
            const int r = ra + lane;
            L.rcnt[r] += int64_t(L.ucnt[L.rbb[r] + L.rnb[r]] - L.ucnt[L.rbb[r]]);
        }
        wave_sync();
        return P;
    }

    // Write the batch left in LDS by batch(ra, rb, ...): rcnt holds each row's
    // first output slot.
    __device__ void write(int ra, int rb, int P) {
        for (int q = lane; q < P; q += kWave) {
            if (L.s_rank[q] == 0xffff) continue;
            const uint32_t j = L.s_j[q];
            const int r = L.ent_row[L.owner[L.s_t[q]]];
            const uint32_t b = L.rbb[r] + uint32_t((uint64_t(j) * L.rscale[r]) >> 32);
            const int64_t p = L.rcnt[r] + int64_t(L.ucnt[b] - L.ucnt[L.rbb[r]]) + L.s_rank[q];
            a.c_ci[p] = int32_t(j);
            Out ov;
            if constexpr (kVal)
                ov = Out(L.s_v[q]);
            else if constexpr (SR == kCount)
                ov = L.s_v[q];
            else
                ov = __int_as_float(L.s_v[q]);
            static_cast<Out*>(a.c_val)[p] = ov;
        }
        // diagonals (lower triangle): the last entry of every non-empty row
        if (LOWER && lane < rb - ra) {
            const int r = ra + lane;
            const int64_t len = L.rp[r + 1] - L.rp[r];
            if (len > 0) {
                const int64_t p = L.rcnt[r] + int64_t(L.ucnt[L.rbb[r] + L.rnb[r]] - L.ucnt[L.rbb[r]]);
                a.c_ci[p] = int32_t(r0 + r);
                Out dv;
                if constexpr (kVal) {
                    double s = 0.0;
                    for (int64_t e = L.rp[r]; e < L.rp[r + 1]; ++e) {
                        const double v = double(static_cast<const In*>(a.val)[e]);
                        s += v * v;
                    }
                    dv = Out(s);
                } else if constexpr (SR == kCount) {
                    dv = int32_t(len);
                } else {
                    dv = jaccard(int32_t(len), len, len);
                }
                static_cast<Out*>(a.c_val)[p] = dv;
            }
        }
        wave_sync();
    }

    __device__ void run(int64_t c) {
        const int R = a.rows_per_chunk;
        r0 = c * R;
        const int nr = int(min(int64_t(R), a.m - r0));
        if (lane <= nr) L.rp[lane] = a.rp[r0 + lane];
        wave_sync();
        if (lane < nr) {
            const int64_t len = L.rp[lane + 1] - L.rp[lane];
            const uint64_t pr = a.prod[r0 + lane];
            const bool light = pr <= uint64_t(kFP) && len <= kFE;
            L.rlight[lane] = light ? 1 : 0;
            L.rprod[lane] = light ? uint16_t(pr) : 0;
            L.rcnt[lane] = light ? ((LOWER && len > 0) ? 1 : 0) : a.heavy_nnz[r0 + lane];
        }
        wave_sync();
        // batches of consecutive light rows (same decision in every lane)
        int nbatch = 0;
        {
            int ra = 0;
            while (ra < nr) {
                while (ra < nr && !L.rlight[ra]) ++ra;
                if (ra >= nr) break;
                int rb = ra;
                int64_t e = 0;
                uint32_t p = 0;
                while (rb < nr && L.rlight[rb]) {
                    const int64_t len = L.rp[rb + 1] - L.rp[rb];
                    if (e + len > kFE || p + L.rprod[rb] > uint32_t(kFP)) break;
                    e += len;
                    p += L.rprod[rb];
                    ++rb;
                }
                if (lane == 0) {
                    L.bra[nbatch] = uint8_t(ra);
                    L.brb[nbatch] = uint8_t(rb);
                }
                ++nbatch;
                ra = rb;
            }
        }
        wave_sync();
        // light rows are written at their upper-bound slots (products + diagonal)
        if (lane < nr) L.rcnt[lane] = a.ubp[r0 + lane];
        wave_sync();
        int64_t cnt = 0;  // exact length of this lane's row
        if (lane < nr) cnt = L.rlight[lane] ? ((LOWER && L.rp[lane + 1] > L.rp[lane]) ? 1 : 0) : a.heavy_nnz[r0 + lane];
        for (int k = 0; k < nbatch; ++k) {
            const int ra = L.bra[k], rb = L.brb[k];
            const int P = batch(ra, rb, false);
            if (lane >= ra && lane < rb)
                cnt += int64_t(L.ucnt[L.rbb[lane] + L.rnb[lane]] - L.ucnt[L.rbb[lane]]);
            write(ra, rb, P);
        }
        if (lane < nr) a.row_cnt[r0 + lane] = cnt;
    }
};

template <int SR, bool LOWER>
__global__ __launch_bounds__(kWave* kWavesF) void fused_kernel(FusedArgs a) {
    using Item = typename ItemOf<SR>::T;
    __shared__ WaveLds<Item> lds[kWavesF];
    WaveLds<Item>& L = lds[threadIdx.x / kWave];
    Chunk<SR, LOWER> ch(a, L);
    const int64_t c = int64_t(blockIdx.x) * kWavesF + threadIdx.x / kWave;
    if (c < a.nchunks) ch.run(c);
}

template <int SR>
void launch(const FusedArgs& a, int grid, hipStream_t s) {
    if (grid <= 0) return;
    if (a.lower)
        fused_kernel<SR, true><<<grid, kWave * kWavesF, 0, s>>>(a);
    else
        fused_kernel<SR, false><<<grid, kWave * kWavesF, 0, s>>>(a);
}

__global__ __launch_bounds__(kBlock) void classify_kernel(const int64_t* __restrict__ rp,
                                                          const unsigned long long* __restrict__ prod, int64_t m,
                                                          bool lower, int32_t* __restrict__ heavy_rows,
                                                          int32_t* heavy_count, unsigned long long* light_cap,
                                                          unsigned long long* prod_sum, int64_t* __restrict__ ub) {
    __shared__ unsigned long long wt[kWavesPerBlock][2];
    unsigned long long cap = 0, ps = 0;
    for (int64_t i = int64_t(blockIdx.x) * kBlock + threadIdx.x; i < m; i += int64_t(gridDim.x) * kBlock) {
        const int64_t len = rp[i + 1] - rp[i];
        const unsigned long long pr = prod[i];
        ps += pr;
        int64_t u = 0;
        if (pr <= (unsigned long long)kFP && len <= kFE) {
            u = int64_t(pr) + ((lower && len > 0) ? 1 : 0);
            cap += u;
        } else {
            heavy_rows[atomicAdd(heavy_count, 1)] = int32_t(i);
        }
        ub[i] = u;
    }
    cap = wave_reduce_sum(cap);
    ps = wave_reduce_sum(ps);
    if (lane_id() == 0) {
        wt[threadIdx.x / kWave][0] = cap;
        wt[threadIdx.x / kWave][1] = ps;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long c = 0, p = 0;
        for (int w = 0; w < kWavesPerBlock; ++w) {
            c += wt[w][0];
            p += wt[w][1];
        }
        if (c) atomicAdd(light_cap, c);
        if (p) atomicAdd(prod_sum, p);
    }
}

}  // namespace

void classify_rows(const int64_t* rp, const unsigned long long* prod, int64_t m, bool lower, int32_t* heavy_rows,
                   int32_t* heavy_count, unsigned long long* light_cap, unsigned long long* prod_sum, int64_t* ub,
                   hipStream_t s) {
    if (m <= 0) return;
    int64_t grid = (m + kBlock - 1) / kBlock;
    if (grid > 1024) grid = 1024;
    classify_kernel<<<unsigned(grid), kBlock, 0, s>>>(rp, prod, m, lower, heavy_rows, heavy_count, light_cap,
                                                      prod_sum, ub);
}

void light_fused(const FusedArgs& a, hipStream_t s) {
    const int grid = int((a.nchunks + kWavesF - 1) / kWavesF);
    if (grid <= 0) return;
    switch (a.sr) {
        case kF64: launch<kF64>(a, grid, s); break;
        case kF32: launch<kF32>(a, grid, s); break;
        case kCount: launch<kCount>(a, grid, s); break;
        default: launch<kJaccard>(a, grid, s); break;
    }
}

int light_fused_waves_per_block() { return kWavesF; }

}  // namespace spsyrk
