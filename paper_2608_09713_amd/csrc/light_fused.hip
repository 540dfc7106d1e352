// Single-pass Gustavson accumulation of the light rows.
//
// Work unit: a chunk of R consecutive rows per wavefront.  Each wavefront
// works alone in its own slice of LDS (no workgroup barriers), in batches of
// consecutive light rows that fit the LDS budget:
//
//   1. partner runs of the batch's entries (written by the column-index
//      build, read in entry order; the next batch's runs are loaded while
//      this batch's keys are in flight);
//   2. products flattened over the entries (the owner entry of every product
//      comes from a scatter of run starts and a max-scan), every key loaded
//      in one round;
//   3. ordered buckets per row (bucket order = column order, about one
//      product per bucket): count, scan, scatter; each small bucket is sorted
//      by (column, product index) in one lane's registers and its equal
//      columns merged (terms summed in product order); the rare large bucket
//      is resolved by the whole wavefront (leader = first product of a
//      column, its rank among the bucket's distinct columns, its value);
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
constexpr int kDealtBelow = 16;      // chunks per launched wavefront below which chunks are dealt out
constexpr int kRunRegs = kFE / kWave;  // partner runs per lane held in registers
constexpr int kSmall = 8;              // buckets up to this size are merged in registers
constexpr int kTBits = 9;              // product index bits in s_t (row above them)
constexpr uint32_t kTMask = (1u << kTBits) - 1u;
// Output tag of a slot once its bucket is merged: the slot's output index in
// the bucket (low kKBits bits) and, for a small bucket, the number of terms
// merged into it (above them; 0 when the value is already final), or 0xffff
// for a slot that writes nothing.
constexpr int kKBits = 9;
constexpr uint32_t kKMask = (1u << kKBits) - 1u;
constexpr uint32_t kNoOut = 0xffffu;
static_assert(kFP <= (1 << kKBits), "an output index must fit kKBits");
static_assert(((kSmall + 1) << kKBits) < int(kNoOut), "a tag must fit 16 bits");
static_assert(kFP <= (1 << kTBits), "product index must fit kTBits");
static_assert(kFR <= (1 << (16 - kTBits)), "chunk row must fit above the product index");


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
    uint32_t rscale[kFR];     // bucket of column j: (j * rscale) >> 32 spreads [0, range) evenly
    uint32_t ent_start[kFE];
    uint16_t ent_len[kFE];
    alignas(4) uint8_t ent_row[kFE];
    int32_t rlen[kFR];        // entries of every row of the batch
    alignas(16) int16_t owner[kFP];
    alignas(16) uint16_t ent_poff[kFE + 1];
    uint32_t s_j[kFP];
    uint16_t s_t[kFP];
    uint16_t s_rank[kFP];     // output tag of every slot (see kKBits)
    uint16_t big[kFP / (kSmall + 1) + 1];  // large buckets of the batch
    uint32_t nbig;
    int64_t rbase[kFR];
    Item s_v[kFP];
    // per bucket (16 bits: every count and offset is at most kFP + kFR)
    alignas(16) uint16_t hist[(kFB + 8) & ~7];
    alignas(16) uint16_t ucnt[kFB + 2];
};
// Two wavefronts' slices must stay within 26880 bytes for six workgroups per
// compute unit (a few bytes more and only five fit, while the occupancy
// query still reports six).
static_assert(sizeof(WaveLds<int32_t>) * kWavesF <= 26880, "LDS slice of the count and Jaccard kernels");

static_assert(kFP + kFR < (1 << 16), "bucket counters are 16 bits");

// atomic add of one to the 16-bit counter h[b] (two counters share a 32-bit
// LDS word; no counter reaches 2^16); returns the old value
__device__ inline uint32_t add16(uint16_t* h, uint32_t b) {
    uint32_t* w = reinterpret_cast<uint32_t*>(h) + (b >> 1);
    const uint32_t sh = (b & 1u) * 16u;
    return (atomicAdd(w, 1u << sh) >> sh) & 0xffffu;
}

// exclusive scan in place of the 16-bit a[0..n) by one wavefront, eight
// elements per lane on 16-byte LDS words (a is 16-byte aligned and holds n
// rounded up to eight; elements past n read as zero); returns the total
__device__ inline uint32_t wave_scan16(uint16_t* a, int n) {
    const int lane = lane_id();
    uint32_t carry = 0;
    for (int base = 0; base < n; base += 8 * kWave) {
        const int i0 = base + 8 * lane;
        uint32_t v[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        if (i0 < n) {
            const uint4 w = *reinterpret_cast<const uint4*>(a + i0);
            const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                v[2 * k] = i0 + 2 * k < n ? (wd[k] & 0xffffu) : 0u;
                v[2 * k + 1] = i0 + 2 * k + 1 < n ? (wd[k] >> 16) : 0u;
            }
        }
        uint32_t sum = 0;
#pragma unroll
        for (int k = 0; k < 8; ++k) sum += v[k];
        const uint32_t inc = wave_inclusive_scan(sum);
        uint32_t off = carry + inc - sum;
        if (i0 < n) {
            uint32_t od[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t lo16 = off;
                off += v[2 * k];
                const uint32_t hi16 = off;
                off += v[2 * k + 1];
                od[k] = (lo16 & 0xffffu) | (hi16 << 16);
            }
            *reinterpret_cast<uint4*>(a + i0) = make_uint4(od[0], od[1], od[2], od[3]);
        }
        carry += __shfl(inc, kWave - 1, kWave);
    }
    wave_sync();
    return carry;
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
    uint32_t lenmax;  // saturated length in a key (Jaccard keys carrying lengths)
    int jbits_right;

    __device__ Chunk(const FusedArgs& a_, WaveLds<Item>& L_) : a(a_), L(L_) {
        lane = lane_id();
        rowmask = a.cx.rowbits >= 32 ? 0xffffffffu : ((1u << a.cx.rowbits) - 1u);
        lenmax = a.cx.lenbits > 0 ? ((a.cx.lenbits >= 32 ? 0xffffffffu : (1u << a.cx.lenbits) - 1u)) : 0u;
        jbits_right = bit_width_u64(a.m_right > 1 ? uint64_t(a.m_right - 1) : 0);
    }

    // Issue the loads of the partner runs of the light rows [ra, rb) (entry
    // lane + kWave * u in rn[u]); they are consumed by the batch's first step.
    __device__ void fetch_runs(int ra, int rb, uint32_t (&rn)[kRunRegs]) {
        const int64_t ebase = L.rp[ra];
        const int ne = int(L.rp[rb] - ebase);
#pragma unroll
        for (int u = 0; u < kRunRegs; ++u) {
            const int x = lane + u * kWave;
            // (a packed word is decoded where the run is used, so that the
            // loads stay in flight)
            rn[u] = x < ne ? a.run.r4[ebase + x] : 0u;
        }
    }

    // Partner runs, buckets, merged columns and per-bucket distinct counts
    // for the light rows [ra, rb), whose runs were fetched into rn.  The
    // batch's columns stay in LDS, grouped by (row, bucket).  The runs of the
    // next batch [na, nb) (if na >= 0) are fetched into rn while the batch's
    // keys are in flight.  Returns the number of products.
    __device__ int batch(int ra, int rb, uint32_t (&rn)[kRunRegs], int na, int nbx) {
        const int64_t ebase = L.rp[ra];
        const int ne = int(L.rp[rb] - ebase);
        const uint32_t* __restrict__ key = a.cx.key;
        // row of every entry: every non-empty row marks its first entry, then
        // a max-scan (four entries per lane, one LDS word)
        static_assert(kFE == 4 * kWave, "one word of entry rows per lane");
        reinterpret_cast<uint32_t*>(L.ent_row)[lane] = 0u;
        wave_sync();
        if (lane < rb - ra) {
            const int r = ra + lane;
            if (L.rp[r + 1] > L.rp[r]) L.ent_row[L.rp[r] - ebase] = uint8_t(r);
        }
#pragma unroll
        for (int u = 0; u < kRunRegs; ++u) {
            const int x = lane + u * kWave;
            if (x < ne) {
                const uint2 r = run_from(a.run, rn[u], ebase + x);
                const uint32_t len = r.y - r.x;
                L.ent_start[x] = r.x;
                L.ent_len[x] = uint16_t(len);
                L.ent_poff[x] = uint16_t(len);
            }
        }
        wave_sync();
        {
            const uint32_t wv = reinterpret_cast<const uint32_t*>(L.ent_row)[lane];
            const uint32_t m0 = wv & 0xffu, m1 = max(m0, (wv >> 8) & 0xffu);
            const uint32_t m2 = max(m1, (wv >> 16) & 0xffu), m3 = max(m2, wv >> 24);
            uint32_t inc = m3;
#pragma unroll
            for (int d = 1; d < kWave; d <<= 1) {
                const uint32_t o = __shfl_up(inc, d, kWave);
                if (lane >= d) inc = max(inc, o);
            }
            uint32_t before = __shfl_up(inc, 1, kWave);
            if (lane == 0) before = 0;
            reinterpret_cast<uint32_t*>(L.ent_row)[lane] = max(before, m0) | (max(before, m1) << 8) |
                                                           (max(before, m2) << 16) | (max(before, m3) << 24);
        }
        wave_sync();
        const int P = int(wave_scan16(L.ent_poff, ne));
        if (lane == 0) L.ent_poff[ne] = uint16_t(P);
        // per-row buckets: one per product (at most one per possible column);
        // bucket of column j = floor(j * nb / range), monotone in j
        const int nrb = rb - ra;
        uint32_t nb = 0;
        if (lane < nrb) {
            const int r = ra + lane;
            L.rlen[r] = int32_t(L.rp[r + 1] - L.rp[r]);
            const int64_t range = LOWER ? (r0 + r) : a.m_right;
            uint64_t want = L.rprod[r] > 0 ? L.rprod[r] : 1;
            if (range > 0 && uint64_t(range) < want) want = uint64_t(range);
            nb = uint32_t(want);
            L.rnb[r] = uint16_t(nb);
            // floor(nb 2^32 / range) rounded down by one more: bucket < nb for
            // every j < range (the quotient's error is far below one); nb <=
            // range, so the scale fits 32 bits
            uint64_t sc = 0;
            if (range > 0) {
                sc = uint64_t(ldexp(double(nb), 32) / double(range));
                sc = sc > 0 ? sc - 1 : 0;
            }
            L.rscale[r] = uint32_t(sc);
        }
        const uint32_t inc = wave_inclusive_scan(nb);
        if (lane < nrb) L.rbb[ra + lane] = uint16_t(inc - nb);
        const uint32_t B = __shfl(inc, kWave - 1, kWave);
        // bucket counters zeroed eight at a time (every bucket's distinct count
        // is set when the buckets are sorted by size)
        for (uint32_t g = lane; 8 * g <= B; g += kWave) reinterpret_cast<uint4*>(L.hist)[g] = make_uint4(0, 0, 0, 0);
        // owner entry of every product: run starts scattered, then a max-scan
        // (eight products per lane, one 16-byte LDS word)
        static_assert(kFP == 8 * kWave, "one 16-byte word of owners per lane");
        reinterpret_cast<uint4*>(L.owner)[lane] = make_uint4(~0u, ~0u, ~0u, ~0u);
        wave_sync();
        for (int x = lane; x < ne; x += kWave)
            if (L.ent_len[x]) L.owner[L.ent_poff[x]] = int16_t(x);
        wave_sync();
        {
            const uint4 wv = reinterpret_cast<const uint4*>(L.owner)[lane];
            const uint32_t wd[4] = {wv.x, wv.y, wv.z, wv.w};
            int o[8];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                o[2 * k] = int(int16_t(wd[k] & 0xffffu));
                o[2 * k + 1] = int(int16_t(wd[k] >> 16));
            }
#pragma unroll
            for (int k = 1; k < 8; ++k) o[k] = max(o[k], o[k - 1]);
            int incm = o[7];
#pragma unroll
            for (int d = 1; d < kWave; d <<= 1) {
                const int u = __shfl_up(incm, d, kWave);
                if (lane >= d) incm = max(incm, u);
            }
            int run = __shfl_up(incm, 1, kWave);
            if (lane == 0) run = -1;
            uint32_t od[4];
#pragma unroll
            for (int k = 0; k < 4; ++k)
                od[k] = (uint32_t(max(o[2 * k], run)) & 0xffffu) | (uint32_t(max(o[2 * k + 1], run)) << 16);
            reinterpret_cast<uint4*>(L.owner)[lane] = make_uint4(od[0], od[1], od[2], od[3]);
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
                    if (!a.cx.lenbits) pv[v] = static_cast<const int32_t*>(a.cx.val)[pos];
                } else if constexpr (kVal) {
                    pv[v] = double(static_cast<const In*>(a.val)[ebase + x]) *
                            double(static_cast<const In*>(a.cx.val)[pos]);
                }
                pb[v] = uint32_t(L.ent_row[x]);
            }
        }
        if (na >= 0) fetch_runs(na, nbx, rn);
#pragma unroll
        for (int v = 0; v < kPV; ++v) {
            const int t = lane + v * kWave;
            if (t < P) {
                const uint32_t j = pj[v] & rowmask;
                if constexpr (SR == kJaccard) {
                    if (a.cx.lenbits) {
                        // the partner's length from its key; saturated: from the row pointers
                        const uint32_t lf = pj[v] >> a.cx.rowbits;
                        pv[v] = lf < lenmax ? int32_t(lf) : int32_t(a.rp_right[j + 1] - a.rp_right[j]);
                    }
                }
                const int r = int(pb[v]);
                pj[v] = j;
                const uint32_t b = L.rbb[r] + __umulhi(j, L.rscale[r]);
                pb[v] = b | (uint32_t(r) << 16);
                add16(L.hist, b);
            }
        }
        wave_sync();
        wave_scan16(L.hist, int(B));
        // scatter into buckets; hist[b] ends as the end of bucket b.  s_t keeps
        // the product index and, above it, the row (one row per bucket)
#pragma unroll
        for (int v = 0; v < kPV; ++v) {
            const int t = lane + v * kWave;
            if (t < P) {
                const uint32_t q = add16(L.hist, pb[v] & 0xffffu);
                // (the owner array is free by now: it keeps every slot's bucket)
                reinterpret_cast<uint16_t*>(L.owner)[q] = uint16_t(pb[v] & 0xffffu);
                L.s_j[q] = pj[v];
                L.s_t[q] = uint16_t(uint32_t(t) | ((pb[v] >> 16) << kTBits));
                if constexpr (SR == kJaccard || kVal) L.s_v[q] = pv[v];
            }
        }
        wave_sync();
        // Buckets by size: empty and single-product buckets are done at once;
        // the others are listed by size class so that every class runs with
        // full lanes.  Small buckets (up to kSmall products), one per lane:
        // sorted by (column, product index) in registers, equal columns merged
        // (terms summed in product order); every column's first product keeps
        // its slot and gets the column's tag in s_rank (term count, index among
        // the bucket's distinct columns), the others are marked as writing
        // nothing; ucnt[b] = distinct columns.  Larger buckets go to the cooperative
        // pass below.  (The entry arrays are free by now and hold the lists.)
        uint16_t* list2 = reinterpret_cast<uint16_t*>(L.ent_start);       // 2 products
        uint16_t* list4 = reinterpret_cast<uint16_t*>(L.ent_start) + kFE;  // 3 or 4
        uint16_t* list8 = L.ent_len;                                       // 5 to 8
        uint32_t n2 = 0, n4 = 0, n8 = 0, nlarge = 0;  // (wave-uniform list lengths)
        const uint64_t lt = lanemask_lt();
        for (uint32_t b0 = 0; b0 < B; b0 += kWave) {
            const uint32_t b = b0 + lane;
            uint32_t sz = 0, lo = 0;
            if (b < B) {
                lo = b ? L.hist[b - 1] : 0u;
                sz = L.hist[b] - lo;
                if (sz == 1) L.s_rank[lo] = uint16_t(1u << kKBits);
                L.ucnt[b] = sz <= 1 ? sz : 0u;
            }
            // wave-aggregated appends
            const uint64_t m2 = __ballot(sz == 2), m4 = __ballot(sz == 3 || sz == 4);
            const uint64_t m8 = __ballot(sz > 4 && sz <= uint32_t(kSmall)), mb = __ballot(sz > uint32_t(kSmall));
            if (sz == 2) list2[n2 + __popcll(m2 & lt)] = uint16_t(b);
            if (sz == 3 || sz == 4) list4[n4 + __popcll(m4 & lt)] = uint16_t(b);
            if (sz > 4 && sz <= uint32_t(kSmall)) list8[n8 + __popcll(m8 & lt)] = uint16_t(b);
            if (sz > uint32_t(kSmall)) L.big[nlarge + __popcll(mb & lt)] = uint16_t(b);
            n2 += __popcll(m2);
            n4 += __popcll(m4);
            n8 += __popcll(m8);
            nlarge += __popcll(mb);
        }
        if (lane == 0) L.nbig = nlarge;
        wave_sync();
        for (uint32_t q = lane; q < n2; q += kWave) {
            const uint32_t b = list2[q];
            const uint32_t lo = b ? L.hist[b - 1] : 0u;
            L.ucnt[b] = merge_two(lo);
        }
        const bool cols32 = !kVal && a.m_right <= (int64_t(1) << 29);
        for (uint32_t q = lane; q < n4; q += kWave) {
            const uint32_t b = list4[q];
            const uint32_t lo = b ? L.hist[b - 1] : 0u, hi = L.hist[b];
            L.ucnt[b] = cols32 ? merge_small_cols<kSmall / 2>(lo, hi - lo) : merge_small<kSmall / 2>(lo, hi - lo);
        }
        for (uint32_t q = lane; q < n8; q += kWave) {
            const uint32_t b = list8[q];
            const uint32_t lo = b ? L.hist[b - 1] : 0u, hi = L.hist[b];
            L.ucnt[b] = cols32 ? merge_small_cols<kSmall>(lo, hi - lo) : merge_small<kSmall>(lo, hi - lo);
        }
        wave_sync();
        // larger buckets, one at a time by the whole wavefront: leaders (first
        // product of each column), their rank among the bucket's distinct
        // columns and their column's value; ucnt[b] = leaders
        const int nbig = int(L.nbig);
        for (int g = 0; g < nbig; ++g) {
            const uint32_t b = L.big[g];
            const uint32_t lo = b ? L.hist[b - 1] : 0u, hi = L.hist[b];
            if (hi - lo <= uint32_t(kWave)) {
                const uint32_t u = merge_wave(lo, hi - lo);
                if (lane == 0) L.ucnt[b] = u;
                wave_sync();
                continue;
            }
            for (uint32_t q = lo + lane; q < hi; q += kWave) {
                const uint32_t j = L.s_j[q];
                const uint32_t t = L.s_t[q] & kTMask;
                bool lead = true;
                for (uint32_t u = lo; u < hi; ++u)
                    if (L.s_j[u] == j && (L.s_t[u] & kTMask) < t) lead = false;
                L.s_rank[q] = lead ? 0 : 0xffff;
            }
            wave_sync();
            uint32_t leaders = 0;
            for (uint32_t q0 = lo; q0 < hi; q0 += kWave) {
                const uint32_t q = q0 + lane;
                bool lead = false;
                Item val = Item(0);
                uint32_t rank = 0;
                if (q < hi && L.s_rank[q] == 0) {
                    lead = true;
                    const uint32_t j = L.s_j[q];
                    const uint32_t t = L.s_t[q] & kTMask;
                    const int r = int(L.s_t[q] >> kTBits);
                    int32_t cnt = 0;
                    for (uint32_t u = lo; u < hi; ++u) {
                        const uint32_t ju = L.s_j[u];
                        rank += (ju < j && L.s_rank[u] != 0xffff) ? 1u : 0u;
                        cnt += ju == j ? 1 : 0;
                    }
                    Item acc = L.s_v[q];
                    if constexpr (kVal) {
                        // terms of column j in product order
                        uint32_t last = t;
                        for (int c = 1; c < cnt; ++c) {
                            uint32_t best = 0xffffffffu, bu = q;
                            for (uint32_t u = lo; u < hi; ++u) {
                                const uint32_t tu = L.s_t[u] & kTMask;
                                if (L.s_j[u] == j && tu > last && tu < best) {
                                    best = tu;
                                    bu = u;
                                }
                            }
                            acc += L.s_v[bu];
                            last = best;
                        }
                    }
                    val = finish(acc, cnt, L.rp[r + 1] - L.rp[r]);
                }
                leaders += uint32_t(__popcll(__ballot(lead)));
                wave_sync();
                if (lead) {
                    L.s_v[q] = val;
                    L.s_rank[q] = uint16_t(rank);
                }
            }
            if (lane == 0) L.ucnt[b] = leaders;
            wave_sync();
        }
        const uint32_t U = wave_scan16(L.ucnt, int(B));
        if (lane == 0) L.ucnt[B] = U;
        wave_sync();
        // first output slot of every row minus its first bucket's offset
        if (lane < nrb) L.rbase[ra + lane] = L.rcnt[ra + lane] - int64_t(L.ucnt[L.rbb[ra + lane]]);
        wave_sync();
        return P;
    }

    // A bucket of up to a wavefront of products at lo, one per lane: a bitonic
    // sort across the lanes by (column, product index, slot), then the first
    // product of every column takes the column's value (terms summed in
    // product order, then finished) and its index among the bucket's distinct
    // columns; the others write nothing.  Returns the distinct columns (the
    // same on every lane).
    __device__ uint32_t merge_wave(uint32_t lo, uint32_t sz) {
        const bool in = uint32_t(lane) < sz;
        uint64_t key = ~uint64_t(0);
        Item v = Item(0);
        if (in) {
            const uint32_t q = lo + uint32_t(lane);
            key = (uint64_t(L.s_j[q]) << 32) | (uint64_t(L.s_t[q] & kTMask) << 6) | uint64_t(lane);
            v = L.s_v[q];
        }
#pragma unroll
        for (int k = 2; k <= kWave; k <<= 1) {
#pragma unroll
            for (int d = k >> 1; d > 0; d >>= 1) {
                const uint64_t pk = (uint64_t(uint32_t(__shfl_xor(uint32_t(key >> 32), d, kWave))) << 32) |
                                    uint64_t(uint32_t(__shfl_xor(uint32_t(key), d, kWave)));
                const Item pv = __shfl_xor(v, d, kWave);
                // keep the smaller key where this lane is the low end of an
                // ascending pair or the high end of a descending one
                const bool keep_min = ((lane & k) == 0) == ((lane & d) == 0);
                if (keep_min ? pk < key : pk > key) {
                    key = pk;
                    v = pv;
                }
            }
        }
        const bool valid = uint32_t(lane) < sz;
        const uint32_t j = uint32_t(key >> 32);
        const uint32_t jp = __shfl_up(j, 1, kWave);
        const bool head = valid && (lane == 0 || jp != j);
        const uint64_t hm = __ballot(head);
        const uint32_t rank = uint32_t(__popcll(hm & lanemask_lt()));
        // the column's terms are this lane's and the next ones up to the next head
        const uint64_t above = lane + 1 < kWave ? hm >> (lane + 1) : 0;
        const uint32_t cnt = above ? uint32_t(__ffsll((long long)above)) : sz - uint32_t(lane);
        Item acc = v;
        if constexpr (kVal) {
            uint32_t cmax = head ? cnt : 1u;
#pragma unroll
            for (int d = 1; d < kWave; d <<= 1) cmax = max(cmax, uint32_t(__shfl_xor(cmax, d, kWave)));
            for (uint32_t c = 1; c < cmax; ++c) {
                const Item w = __shfl_down(v, c, kWave);
                if (head && c < cnt) acc += w;
            }
        }
        if (valid) {
            const uint32_t q = lo + uint32_t(key & 63u);
            if (head) {
                const int r = int(L.s_t[q] >> kTBits);
                L.s_v[q] = finish(acc, int32_t(cnt), L.rp[r + 1] - L.rp[r]);
                L.s_rank[q] = uint16_t(rank);
            } else {
                L.s_rank[q] = uint16_t(kNoOut);
            }
        }
        wave_sync();
        return uint32_t(__popcll(hm));
    }

    // Sort the sz (<= N) products at [lo, lo + sz) by (column, product index)
    // in registers, each key carrying its slot.  The first product of every
    // column takes the column's tag (term count, index among the bucket's
    // distinct columns) and, for plus-times with several terms, their sum in
    // product order; the other products of the column write nothing.  Returns
    // the number of distinct columns.
    template <int N>
    __device__ uint32_t merge_small(uint32_t lo, uint32_t sz) {
        static_assert(N <= 16, "slots in four bits");
        uint64_t k[N];
        Item v[N];
#pragma unroll
        for (int u = 0; u < N; ++u) {
            const bool in = uint32_t(u) < sz;
            k[u] = in ? ((((uint64_t(L.s_j[lo + u]) << 16) | L.s_t[lo + u]) << 4) | uint64_t(u)) : ~uint64_t(0);
            v[u] = in ? L.s_v[lo + u] : Item(0);
        }
        if constexpr (N == 4) {
            cswap(k, v, 0, 1); cswap(k, v, 2, 3); cswap(k, v, 0, 2); cswap(k, v, 1, 3); cswap(k, v, 1, 2);
        } else {
            static_assert(N == 8, "networks for 4 and 8 products");
            cswap(k, v, 0, 1); cswap(k, v, 2, 3); cswap(k, v, 4, 5); cswap(k, v, 6, 7);
            cswap(k, v, 0, 2); cswap(k, v, 1, 3); cswap(k, v, 4, 6); cswap(k, v, 5, 7);
            cswap(k, v, 1, 2); cswap(k, v, 5, 6); cswap(k, v, 0, 4); cswap(k, v, 3, 7);
            cswap(k, v, 1, 5); cswap(k, v, 2, 6);
            cswap(k, v, 1, 4); cswap(k, v, 3, 6);
            cswap(k, v, 2, 4); cswap(k, v, 3, 5);
            cswap(k, v, 3, 4);
        }
        uint32_t d = 0;
        uint32_t gj = uint32_t(k[0] >> 20);
        uint32_t gs = uint32_t(k[0] & 15u);
        Item acc = v[0];
        uint32_t cnt = 1;
#pragma unroll
        for (int u = 1; u <= N; ++u) {
            const bool in = uint32_t(u) < sz;
            const uint64_t ku = k[u < N ? u : 0];
            const uint32_t j = in ? uint32_t(ku >> 20) : 0u;
            if (in && j == gj) {
                ++cnt;
                if constexpr (kVal) acc += v[u < N ? u : 0];
                L.s_rank[lo + uint32_t(ku & 15u)] = uint16_t(kNoOut);
            } else if (uint32_t(u) <= sz) {
                // the group of gj ends
                L.s_rank[lo + gs] = uint16_t((cnt << kKBits) | d);
                if constexpr (kVal)
                    if (cnt > 1) L.s_v[lo + gs] = acc;
                ++d;
                if (in) {
                    gj = j;
                    gs = uint32_t(ku & 15u);
                    acc = v[u < N ? u : 0];
                    cnt = 1;
                }
            }
        }
        return d;
    }

    // The same for counts and Jaccard values, whose terms need no order: the
    // keys are (column, slot) in 32 bits (columns below 2^29), sorted with
    // min/max pairs, and only the columns are loaded.  Any product of a
    // column may take its tag: the output is the same.
    template <int N>
    __device__ uint32_t merge_small_cols(uint32_t lo, uint32_t sz) {
        static_assert(N <= 8, "slots in three bits");
        uint32_t k[N];
#pragma unroll
        for (int u = 0; u < N; ++u) k[u] = uint32_t(u) < sz ? ((L.s_j[lo + u] << 3) | uint32_t(u)) : 0xffffffffu;
        auto cs = [&](int x, int y) {
            const uint32_t a = min(k[x], k[y]), b = max(k[x], k[y]);
            k[x] = a;
            k[y] = b;
        };
        if constexpr (N == 4) {
            cs(0, 1); cs(2, 3); cs(0, 2); cs(1, 3); cs(1, 2);
        } else {
            static_assert(N == 8, "networks for 4 and 8 products");
            cs(0, 1); cs(2, 3); cs(4, 5); cs(6, 7);
            cs(0, 2); cs(1, 3); cs(4, 6); cs(5, 7);
            cs(1, 2); cs(5, 6); cs(0, 4); cs(3, 7);
            cs(1, 5); cs(2, 6);
            cs(1, 4); cs(3, 6);
            cs(2, 4); cs(3, 5);
            cs(3, 4);
        }
        uint32_t d = 0, gj = k[0] >> 3, gs = k[0] & 7u, cnt = 1;
#pragma unroll
        for (int u = 1; u <= N; ++u) {
            const bool in = uint32_t(u) < sz;
            const uint32_t ku = k[u < N ? u : 0];
            const uint32_t j = in ? ku >> 3 : 0u;
            if (in && j == gj) {
                ++cnt;
                L.s_rank[lo + (ku & 7u)] = uint16_t(kNoOut);
            } else if (uint32_t(u) <= sz) {
                L.s_rank[lo + gs] = uint16_t((cnt << kKBits) | d);
                ++d;
                if (in) {
                    gj = j;
                    gs = ku & 7u;
                    cnt = 1;
                }
            }
        }
        return d;
    }

    // A bucket of two products at lo.  Distinct columns keep their slots and
    // get their output order in their tags; equal columns merge into the
    // first slot (terms in product order).  Returns the distinct columns.
    __device__ uint32_t merge_two(uint32_t lo) {
        const uint32_t j0 = L.s_j[lo], j1 = L.s_j[lo + 1];
        if (j0 != j1) {
            const uint32_t f = j1 < j0 ? 1u : 0u;
            L.s_rank[lo] = uint16_t((1u << kKBits) | f);
            L.s_rank[lo + 1] = uint16_t((1u << kKBits) | (f ^ 1u));
            return 2;
        }
        if constexpr (kVal) {
            const uint32_t t0 = L.s_t[lo], t1 = L.s_t[lo + 1];
            const Item v0 = L.s_v[lo], v1 = L.s_v[lo + 1];
            L.s_v[lo] = t0 < t1 ? v0 + v1 : v1 + v0;
        }
        L.s_rank[lo] = uint16_t(2u << kKBits);
        L.s_rank[lo + 1] = uint16_t(kNoOut);
        return 1;
    }

    // value of a merged column: the sum (plus-times), the count, or the
    // Jaccard bits from the count and the two row lengths (with packed
    // staging: the count and the partner's length, cnt * pack_r2 + |S(j)|,
    // for the compaction to finish)
    __device__ Item finish(Item acc, int32_t cnt, int64_t len_i) const {
        if constexpr (kVal)
            return acc;
        else if constexpr (SR == kCount)
            return cnt;
        else
            return a.pack_rr ? int32_t(uint32_t(cnt) * a.pack_r2 + uint32_t(acc))
                             : __float_as_int(jaccard(cnt, len_i, acc));
    }

    template <int N>
    __device__ static void cswap(uint64_t (&k)[N], Item (&v)[N], int x, int y) {
        const bool sw = k[y] < k[x];
        const uint64_t kx = sw ? k[y] : k[x], ky = sw ? k[x] : k[y];
        const Item vx = sw ? v[y] : v[x], vy = sw ? v[x] : v[y];
        k[x] = kx;
        k[y] = ky;
        v[x] = vx;
        v[y] = vy;
    }

    // Write the batch left in LDS by batch(ra, rb, ...) (nprod products):
    // rcnt holds each row's first output slot, rbase that slot minus the
    // offset of the row's first bucket.
    __device__ void write(int ra, int rb, int nprod) {
        // outputs in slot order (about output order), each found from its
        // slot's bucket: consecutive lanes write consecutive slots of a row
        const uint16_t* sbk = reinterpret_cast<const uint16_t*>(L.owner);
        for (int q = lane; q < nprod; q += kWave) {
            const uint32_t tag = L.s_rank[q];
            if (tag == kNoOut) continue;
            const uint32_t b = sbk[q];
            const int r = int(L.s_t[q] >> kTBits);
            Item v = L.s_v[q];
            const uint32_t cnt = tag >> kKBits;
            if (cnt) v = finish(v, int32_t(cnt), L.rlen[r]);
            emit(L.rbase[r] + int64_t(uint32_t(L.ucnt[b]) + (tag & kKMask)), L.s_j[q], v);
        }
        // diagonals (lower triangle): the last entry of every non-empty row
        if (LOWER && lane < rb - ra) {
            const int r = ra + lane;
            const int64_t len = L.rp[r + 1] - L.rp[r];
            if (len > 0) {
                const int64_t p = L.rcnt[r] + int64_t(L.ucnt[L.rbb[r] + L.rnb[r]] - L.ucnt[L.rbb[r]]);
                Item dv;
                if constexpr (kVal) {
                    double s = 0.0;
                    for (int64_t e = L.rp[r]; e < L.rp[r + 1]; ++e) {
                        const double v = double(static_cast<const In*>(a.val)[e]);
                        s += v * v;
                    }
                    dv = s;
                } else {
                    dv = finish(Item(len), int32_t(len), len);  // |S(i) and S(i)| = |S(i)|
                }
                emit(p, uint32_t(r0 + r), dv);
            }
        }
        wave_sync();
    }

    __device__ void emit(int64_t p, uint32_t j, Item v) {
        if constexpr (!kVal) {
            if (a.pack_rr) {  // one staged word: column and packed value
                reinterpret_cast<uint32_t*>(a.c_ci)[p] = j * a.pack_rr + uint32_t(v);
                return;
            }
        }
        a.c_ci[p] = int32_t(j);
        Out ov;
        if constexpr (kVal)
            ov = Out(v);
        else if constexpr (SR == kCount)
            ov = v;
        else
            ov = __int_as_float(v);
        static_cast<Out*>(a.c_val)[p] = ov;
    }

    // A chunk's row pointers, product counts and staging slots (lane = row),
    // loaded in one round, ahead of the chunk.
    struct Head {
        int64_t rpv = 0, ubv = 0;
        uint64_t pr = 0;
    };
    __device__ Head head(int64_t c) const {
        const int R = a.rows_per_chunk;
        const int64_t rs = c * R;
        const int nr = int(min(int64_t(R), a.m - rs));
        Head h;
        if (lane <= nr) h.rpv = a.rp[rs + lane];
        if (lane < nr) {
            h.pr = a.prod[rs + lane];
            h.ubv = a.ubp[rs + lane];
        }
        return h;
    }

    __device__ void run(int64_t c, const Head& h) {
        const int R = a.rows_per_chunk;
        r0 = c * R;
        const int nr = int(min(int64_t(R), a.m - r0));
        const int64_t rpv = h.rpv, ubv = h.ubv;
        const uint64_t pr = h.pr;
        if (lane <= nr) L.rp[lane] = rpv;
        wave_sync();
        int64_t len = 0;
        bool light = false;
        const int64_t rpn = __shfl_down(rpv, 1, kWave);  // row pointer after this lane's row
        if (lane < nr) {
            len = rpn - rpv;
            light = pr <= uint64_t(kFP) && len <= kFE;
            L.rprod[lane] = light ? uint16_t(pr) : 0;
            // light rows are written at their upper-bound slots (products + diagonal)
            L.rcnt[lane] = ubv;
        }
        // batches of consecutive light rows, cut greedily: a batch opened at
        // row ra takes the following light rows while its entries and products
        // fit the LDS budget; every lane tests its own row against the prefix
        // sums at ra, and the batch ends at the first row that fails.  Lane k
        // keeps batch k's rows (ra | rb << 8).
        const uint64_t lightmask = __ballot(lane < nr && light);
        const uint32_t mypr = (lane < nr && light) ? uint32_t(pr) : 0u;
        const uint32_t pinc = wave_inclusive_scan(mypr);
        const uint32_t pexc = pinc - mypr;
        int nbatch = 0;
        uint32_t mybatch = 0;
        for (uint64_t rest = lightmask; rest;) {
            const int ra = __ffsll((unsigned long long)rest) - 1;
            const int64_t ea = int64_t(uint64_t(uint32_t(__builtin_amdgcn_readlane(int(uint32_t(rpv)), ra))) |
                                       (uint64_t(uint32_t(__builtin_amdgcn_readlane(int(uint32_t(uint64_t(rpv) >> 32)), ra))) << 32));
            const uint32_t pa = uint32_t(__builtin_amdgcn_readlane(int(pexc), ra));
            const bool ok = lane >= ra && lane < nr && light && rpn - ea <= kFE && pinc - pa <= uint32_t(kFP);
            const uint64_t okm = __ballot(ok) >> ra;
            const int rb = ra + __ffsll((unsigned long long)~okm) - 1;
            if (lane == nbatch) mybatch = uint32_t(ra) | (uint32_t(rb) << 8);
            ++nbatch;
            rest = lightmask & (~uint64_t(0) << rb);
        }
        wave_sync();
        int64_t cnt = 0;  // exact length of this lane's row
        if (lane < nr) cnt = light ? ((LOWER && len > 0) ? 1 : 0) : a.heavy_nnz[r0 + lane];
        uint32_t rn[kRunRegs];
        uint32_t bk = nbatch > 0 ? uint32_t(__builtin_amdgcn_readlane(int(mybatch), 0)) : 0u;
        if (nbatch > 0) fetch_runs(int(bk & 0xffu), int(bk >> 8), rn);
        for (int k = 0; k < nbatch; ++k) {
            const int ra = int(bk & 0xffu), rb = int(bk >> 8);
            const bool more = k + 1 < nbatch;
            const uint32_t bn = more ? uint32_t(__builtin_amdgcn_readlane(int(mybatch), k + 1)) : 0u;
            const int P = batch(ra, rb, rn, more ? int(bn & 0xffu) : -1, more ? int(bn >> 8) : 0);
            bk = bn;
            if (lane >= ra && lane < rb)
                cnt += int64_t(L.ucnt[L.rbb[lane] + L.rnb[lane]] - L.ucnt[L.rbb[lane]]);
            write(ra, rb, P);
        }
        if (lane < nr) a.row_cnt[r0 + lane] = cnt;
    }
};

template <int SR, bool LOWER>
// (plus-times: at most 168 VGPRs, three wavefronts per SIMD)
__global__ __launch_bounds__(kWave* kWavesF) __attribute__((amdgpu_waves_per_eu(SR == kF64 || SR == kF32 ? 3 : 1)))
void fused_kernel(FusedArgs a) {
    using Item = typename ItemOf<SR>::T;
    __shared__ WaveLds<Item> lds[kWavesF];
    WaveLds<Item>& L = lds[threadIdx.x / kWave];
    Chunk<SR, LOWER> ch(a, L);
    // Persistent wavefronts.  With few chunks per launched wavefront the
    // chunks are dealt out in turn (c, c + stride, ...).  With many, the
    // wavefronts take runs of consecutive chunks from a counter, so that
    // every wavefront the device holds keeps busy however many of the
    // launched ones are resident at once and however the chunks' costs vary:
    // a run is a quarter of the chunks left per launched wavefront (as last
    // seen), at least one, so the runs shrink towards the end.  The next
    // chunk is taken and its head loaded while the current chunk runs.
    const int lane = lane_id();
    if (blockIdx.x == 0 && threadIdx.x == 0) a.row_cnt[a.m] = 0;  // (the scan's last input)
    const int64_t nwaves = int64_t(gridDim.x) * kWavesF;
    const bool dealt = a.nchunks < kDealtBelow * nwaves;
    int64_t seen = 0, rend = 0;
    auto take = [&]() -> int64_t {
        if (dealt) {
            const int64_t c = seen ? rend + nwaves - 1 : int64_t(blockIdx.x) * kWavesF + threadIdx.x / kWave;
            seen = 1;
            rend = c + 1;
            return c;
        }
        int64_t g = (a.nchunks - seen) / (4 * nwaves);
        g = g < 1 ? 1 : g;
        unsigned long long c0 = 0;
        if (lane == 0) c0 = atomicAdd(a.chunk_counter, (unsigned long long)g);
        const int64_t c = int64_t(__shfl(c0, 0, kWave));
        seen = c + g;
        rend = c + g;
        return c;
    };
    int64_t c = take();
    if (c >= a.nchunks) return;
    auto h = ch.head(c);
    while (true) {
        const int64_t cn = c + 1 < rend ? c + 1 : take();
        decltype(h) hn;
        if (cn < a.nchunks) hn = ch.head(cn);
        ch.run(c, h);
        if (cn >= a.nchunks) break;
        c = cn;
        h = hn;
    }
}

// Workgroups resident on the whole device at once (at least one).
template <typename K>
int resident_groups(K kernel) {
    int dev = 0, cus = 0, per = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 1;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 1;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kernel, kWave * kWavesF, 0) != hipSuccess) return 1;
    const int g = cus * per;
    return g > 0 ? g : 1;
}

template <int SR>
void launch(const FusedArgs& a, int grid, hipStream_t s) {
    if (grid <= 0) return;
    if (a.lower) {
        static const int res = resident_groups(fused_kernel<SR, true>);
        fused_kernel<SR, true><<<grid < res ? grid : res, kWave * kWavesF, 0, s>>>(a);
    } else {
        static const int res = resident_groups(fused_kernel<SR, false>);
        fused_kernel<SR, false><<<grid < res ? grid : res, kWave * kWavesF, 0, s>>>(a);
    }
}

__global__ __launch_bounds__(kBlock) void classify_kernel(const int64_t* __restrict__ rp,
                                                          const unsigned long long* __restrict__ prod, int64_t m,
                                                          bool lower, int32_t* __restrict__ heavy_rows,
                                                          int32_t* heavy_count, unsigned long long* light_cap,
                                                          unsigned long long* prod_sum, int64_t* __restrict__ ub,
                                                          unsigned long long* maxlen) {
    __shared__ unsigned long long wt[kWavesPerBlock][3];
    unsigned long long cap = 0, ps = 0, ml = 0;
    for (int64_t i = int64_t(blockIdx.x) * kBlock + threadIdx.x; i < m; i += int64_t(gridDim.x) * kBlock) {
        const int64_t len = rp[i + 1] - rp[i];
        const unsigned long long pr = prod[i];
        ps += pr;
        ml = max(ml, (unsigned long long)len);
        int64_t u = 0;
        if (pr <= (unsigned long long)kFP && len <= kFE) {
            u = int64_t(pr) + ((lower && len > 0) ? 1 : 0);
            cap += u;
        } else {
            heavy_rows[atomicAdd(heavy_count, 1)] = int32_t(i);
        }
        ub[i] = u;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) ub[m] = 0;  // (the scan's last input)
    cap = wave_reduce_sum(cap);
    ps = wave_reduce_sum(ps);
    ml = wave_reduce_max(ml);
    if (lane_id() == 0) {
        wt[threadIdx.x / kWave][0] = cap;
        wt[threadIdx.x / kWave][1] = ps;
        wt[threadIdx.x / kWave][2] = ml;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long c = 0, p = 0, l = 0;
        for (int w = 0; w < kWavesPerBlock; ++w) {
            c += wt[w][0];
            p += wt[w][1];
            l = max(l, wt[w][2]);
        }
        if (c) atomicAdd(light_cap, c);
        if (p) atomicAdd(prod_sum, p);
        if (l && maxlen) atomicMax(maxlen, l);
    }
}

}  // namespace

void classify_rows(const int64_t* rp, const unsigned long long* prod, int64_t m, bool lower, int32_t* heavy_rows,
                   int32_t* heavy_count, unsigned long long* light_cap, unsigned long long* prod_sum, int64_t* ub,
                   hipStream_t s, unsigned long long* maxlen) {
    if (m <= 0) return;
    int64_t grid = (m + kBlock - 1) / kBlock;
    if (grid > 1024) grid = 1024;
    classify_kernel<<<unsigned(grid), kBlock, 0, s>>>(rp, prod, m, lower, heavy_rows, heavy_count, light_cap,
                                                      prod_sum, ub, maxlen);
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
