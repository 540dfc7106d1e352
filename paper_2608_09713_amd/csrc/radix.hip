// Stable least-significant-digit radix sort of (key, row, value) records by
// key bits, at most 8 bits per pass (the key's bits spread evenly over the
// passes).  Used to group the entries of a CSR matrix by column while keeping
// rows ascending inside each column (the input is in row order and every pass
// is stable).
//
// Per pass: (1) per-tile digit histograms, (2) exclusive scan of the
// digit-major (digit, tile) count matrix, (3) stable scatter: every wave ranks
// its contiguous kSeg-record segment with ballot-based digit matching and
// per-wave LDS counters, the tile is reordered through LDS, then written out
// so that consecutive threads store consecutive addresses of a digit's run.
#include <algorithm>
#include <cstdlib>
#include <type_traits>

#include "common.h"
#include "internal.h"

namespace spsyrk {
namespace {

constexpr int kRBits = 8;
constexpr int kDigits = 1 << kRBits;
constexpr int kRItems = 12;
constexpr int kRTile = kBlock * kRItems;  // records per tile
static_assert(kRTile == kRadixTile, "the validation counts the first pass's digits over the same tiles");
constexpr int kSeg = kWave * kRItems;     // records per wave

template <int VB>
struct ValT {
    using T = uint32_t;
};
template <>
struct ValT<8> {
    using T = uint64_t;
};

__global__ __launch_bounds__(kBlock) void radix_hist(const uint32_t* __restrict__ keys, int64_t n, int shift,
                                                     uint32_t mask, uint32_t* __restrict__ hist, int64_t ntiles) {
    // consecutive tiles on one XCD, so that one L2 gathers their counts'
    // 4-byte writes (hist is digit-major: tile t of digit d at d * ntiles + t)
    const int64_t per = (ntiles + kXcds - 1) / kXcds;
    const int64_t tile = int64_t(blockIdx.x % kXcds) * per + blockIdx.x / kXcds;
    if (tile >= ntiles) return;
    // one sub-histogram per wavefront keeps the LDS atomics of different
    // wavefronts apart
    __shared__ uint32_t cnt[kWavesPerBlock][kDigits];
    const int w = threadIdx.x / kWave;
#pragma unroll
    for (int q = 0; q < kWavesPerBlock; ++q) cnt[q][threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = tile * kRTile;
    if (base + kRTile <= n && (reinterpret_cast<uintptr_t>(keys) & 15) == 0) {
        // whole tile, 16-byte loads (the tile starts at a multiple of 16 bytes)
        uint4 kv[kRItems / 4];
#pragma unroll
        for (int k = 0; k < kRItems / 4; ++k)
            kv[k] = reinterpret_cast<const uint4*>(keys + base)[k * kBlock + threadIdx.x];
#pragma unroll
        for (int k = 0; k < kRItems / 4; ++k) {
            atomicAdd(&cnt[w][(kv[k].x >> shift) & mask], 1u);
            atomicAdd(&cnt[w][(kv[k].y >> shift) & mask], 1u);
            atomicAdd(&cnt[w][(kv[k].z >> shift) & mask], 1u);
            atomicAdd(&cnt[w][(kv[k].w >> shift) & mask], 1u);
        }
    } else {
        uint32_t kk[kRItems];
#pragma unroll
        for (int k = 0; k < kRItems; ++k) {
            const int64_t i = base + int64_t(k) * kBlock + threadIdx.x;
            kk[k] = i < n ? keys[i] : 0xffffffffu;
        }
#pragma unroll
        for (int k = 0; k < kRItems; ++k) {
            const int64_t i = base + int64_t(k) * kBlock + threadIdx.x;
            if (i < n) atomicAdd(&cnt[w][(kk[k] >> shift) & mask], 1u);
        }
    }
    __syncthreads();
    uint32_t t = 0;
#pragma unroll
    for (int q = 0; q < kWavesPerBlock; ++q) t += cnt[q][threadIdx.x];
    hist[int64_t(threadIdx.x) * ntiles + tile] = t;
}

constexpr int kRowWin = 1024;

__device__ inline int64_t last_leq_i64(const int64_t* a, int64_t lo, int64_t hi, int64_t x) {
    while (lo < hi) {
        const int64_t mid = (lo + hi + 1) >> 1;
        if (a[mid] <= x)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

// Where a pass takes its records from (SRC) and puts them (OUT).
//  kSrcArrays: key, row and value arrays.
//  kSrcCsr: straight from a CSR matrix: key = column, row from the row
//    pointers (rp, m), value = the entry's index (VB 4), or with val_in the
//    entry's value (VB 4 or 8, read from val_in in entry order).  With
//    lenbits > 0 the row field also carries the row's length, saturated at
//    2^lenbits - 1, above its low rowbits bits.
//  kSrcSlab: a mirror slab's strict-lower entries, record p of row r (rows
//    from the record pointers rp = rec_rp) being entry p + sl.row_off[r] of
//    C_L: key = column - sl.c0, row = r, value = the
//    entry's value.
//  kOutArrays: key, row and value arrays in the pass's order.
//  kOutPlace (last pass of a mirror slab): keys to key_out; the row and
//    value of the record at sorted position q to the full rows, at
//    sl.before + q + sl.rp[sl.c0 + key + 1] (its column's lower part, then
//    the strict entries of the column in row order).
constexpr int kSrcArrays = 0, kSrcCsr = 1, kSrcSlab = 2;
constexpr int kOutArrays = 0, kOutPlace = 1;

// rowof[i] = the row of record base + i of a tile of a record structure with
// row pointers rp (rows [rlo, rhi] span the tile, rlo holding its first
// record): every row that starts inside the tile marks its first record,
// then a running maximum over the tile.  The rows are walked one by one, not
// staged, so any number of empty rows may lie between (each row pointer is
// read by about one tile).  Called by all threads; wt: kWavesPerBlock words.
__device__ inline void tile_rows_mark(const int64_t* __restrict__ rp, int64_t rlo, int64_t rhi, int64_t base,
                                      uint32_t* rowof, uint32_t* wt) {
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    for (int i = threadIdx.x; i < kRTile; i += kBlock) rowof[i] = uint32_t(rlo);
    __syncthreads();
    for (int64_t k = rlo + 1 + threadIdx.x; k <= rhi; k += kBlock) {
        const int64_t a = rp[k];
        if (a - base < kRTile && rp[k + 1] > a) rowof[a - base] = uint32_t(k);
    }
    __syncthreads();
    uint32_t run_max = 0;
#pragma unroll
    for (int k = 0; k < kRItems; ++k) run_max = max(run_max, rowof[threadIdx.x * kRItems + k]);
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
    for (int k = 0; k < kRItems; ++k) {
        before = max(before, rowof[threadIdx.x * kRItems + k]);
        rowof[threadIdx.x * kRItems + k] = before;
    }
    __syncthreads();
}

// Digit counts of the first pass over a mirror slab (kSrcSlab): every key
// read through its record's row.
__global__ __launch_bounds__(kBlock) void radix_hist_slab(int64_t n, uint32_t mask, uint32_t* __restrict__ hist,
                                                          int64_t ntiles, const int64_t* __restrict__ rp, int64_t m,
                                                          const int64_t* __restrict__ trow, SlabIo sl) {
    __shared__ uint32_t cnt[kWavesPerBlock][kDigits];
    __shared__ uint32_t rowof[kRTile];
    __shared__ uint32_t wt[kWavesPerBlock];
    __shared__ int64_t rb[2];
    const int64_t per = (ntiles + kXcds - 1) / kXcds;  // (tiles placed as in radix_hist)
    const int64_t tile = int64_t(blockIdx.x % kXcds) * per + blockIdx.x / kXcds;
    if (tile >= ntiles) return;
    const int w = threadIdx.x / kWave;
#pragma unroll
    for (int q = 0; q < kWavesPerBlock; ++q) cnt[q][threadIdx.x] = 0;
    const int64_t base = tile * kRTile;
    if (threadIdx.x == 0) {
        rb[0] = trow[tile];
        rb[1] = base + kRTile < n ? trow[tile + 1] : last_leq_i64(rp, trow[tile], m, n - 1);
    }
    __syncthreads();
    tile_rows_mark(rp, rb[0], rb[1], base, rowof, wt);
    uint32_t key[kRItems];
#pragma unroll
    for (int k = 0; k < kRItems; ++k) {
        const int64_t idx = base + int64_t(k) * kBlock + threadIdx.x;
        key[k] = 0;
        if (idx < n) {
            const int64_t r = rowof[idx - base];
            key[k] = uint32_t(int64_t(sl.ci[idx + sl.row_off[r]]) - sl.c0);
        }
    }
#pragma unroll
    for (int k = 0; k < kRItems; ++k)
        if (base + int64_t(k) * kBlock + threadIdx.x < n) atomicAdd(&cnt[w][key[k] & mask], 1u);
    __syncthreads();
    uint32_t t = 0;
#pragma unroll
    for (int q = 0; q < kWavesPerBlock; ++q) t += cnt[q][threadIdx.x];
    hist[int64_t(threadIdx.x) * ntiles + tile] = t;
}

template <int VB, int SRC, int OUT = kOutArrays>
__global__ __launch_bounds__(kBlock) void radix_scatter(const uint32_t* __restrict__ key_in,
                                                        const uint32_t* __restrict__ row_in,
                                                        const typename ValT<VB>::T* __restrict__ val_in,
                                                        uint32_t* __restrict__ key_out, uint32_t* __restrict__ row_out,
                                                        typename ValT<VB>::T* __restrict__ val_out, int64_t n, int shift,
                                                        uint32_t mask, const uint32_t* __restrict__ offs,
                                                        int64_t ntiles, const int64_t* __restrict__ rp, int64_t m,
                                                        const int64_t* __restrict__ trow, int rowbits, int lenbits,
                                                        SlabIo sl) {
    using V = typename ValT<VB>::T;
    constexpr bool FIRST = SRC != kSrcArrays;  // records derived from a row structure
    // consecutive tiles on one XCD (workgroups go round-robin over the XCDs),
    // so the partial lines where their digit runs meet merge in one L2
    const int64_t per = (ntiles + kXcds - 1) / kXcds;
    const int64_t tile = int64_t(blockIdx.x % kXcds) * per + blockIdx.x / kXcds;
    if (tile >= ntiles) return;
    __shared__ int64_t rwin[SRC == kSrcCsr ? kRowWin + 1 : 1];
    __shared__ int64_t rbounds[2];
    __shared__ uint32_t wcnt[kWavesPerBlock][kDigits];
    __shared__ int64_t gofs[kDigits];  // global position of the tile's digit run minus its tile start
    __shared__ uint32_t wt[kWavesPerBlock];
    // the tile is reordered through one buffer, a field at a time
    __shared__ V ex[kRTile];
    __shared__ uint8_t dig[kRTile];
    __shared__ uint16_t kslot[OUT == kOutPlace ? kRTile : 1];  // key of every slot (keys below 2^16)

    const int w = threadIdx.x / kWave;
    const int lane = lane_id();
    const int64_t base = tile * kRTile;
    const int64_t segbase = base + int64_t(w) * kSeg;
    // the keys (the column ids in the first pass) are read once, with
    // streaming loads so that they do not push the tile's partly written
    // output lines out of L2, and first, so that they arrive while the tile
    // is set up (a slab's keys are read through its rows, further below)
    uint32_t kr[kRItems];
    if constexpr (SRC != kSrcSlab) {
#pragma unroll
        for (int k = 0; k < kRItems; ++k) {
            const int64_t idx = segbase + int64_t(k) * kWave + lane;
            kr[k] = idx < n ? __builtin_nontemporal_load(key_in + idx) : 0u;
        }
    }
#pragma unroll
    for (int q = 0; q < kWavesPerBlock; ++q) wcnt[q][threadIdx.x] = 0;
    __syncthreads();

    int64_t rlo = 0, rhi = 0;
    bool rstaged = false;
    if constexpr (FIRST) {
        if (threadIdx.x == 0) {
            // rows of the tile's first entry and (at most one row past the
            // tile) of its end, from the tile table; the last tile searches,
            // and so does a tile the table leaves out (-1: a table written
            // by the validation skips the tiles deep inside very long rows)
            int64_t lo = trow[tile];
            if (lo < 0) lo = last_leq_i64(rp, 0, m, base);
            int64_t hi = base + kRTile < n ? trow[tile + 1] : -1;
            if (hi < 0) hi = last_leq_i64(rp, lo, m, base + kRTile < n ? base + kRTile : n - 1);
            rbounds[0] = lo;
            rbounds[1] = hi;
        }
        __syncthreads();
        rlo = rbounds[0];
        rhi = rbounds[1];
        rstaged = SRC == kSrcCsr && rhi - rlo + 2 <= kRowWin + 1;
        if constexpr (SRC == kSrcSlab) tile_rows_mark(rp, rlo, rhi, base, reinterpret_cast<uint32_t*>(ex), wt);
        if (rstaged) {
            for (int64_t k = threadIdx.x; k < rhi - rlo + 2; k += kBlock) rwin[k] = rp[rlo + k];
            // window row of every tile position (in the exchange buffer, free
            // until the records are reordered): every non-empty row marks its
            // first position, then a max-scan over the tile
            uint32_t* rowof = reinterpret_cast<uint32_t*>(ex);
            for (int i = threadIdx.x; i < kRTile; i += kBlock) rowof[i] = 0;
            __syncthreads();
            for (int64_t k = 1 + threadIdx.x; k <= rhi - rlo; k += kBlock)
                if (rwin[k] < rwin[k + 1] && rwin[k] - base < kRTile) rowof[rwin[k] - base] = uint32_t(k);
            __syncthreads();
            uint32_t run_max = 0;
#pragma unroll
            for (int k = 0; k < kRItems; ++k) run_max = max(run_max, rowof[threadIdx.x * kRItems + k]);
            // exclusive max over the preceding threads
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
            for (int k = 0; k < kRItems; ++k) {
                before = max(before, rowof[threadIdx.x * kRItems + k]);
                rowof[threadIdx.x * kRItems + k] = before;
            }
        }
        __syncthreads();
    }
    // keys and tile positions stay in registers; the first pass also keeps
    // its row fields (computed from the LDS window, which the exchange
    // buffer overwrites), other passes load rows and values only when they
    // are exchanged (fewer registers, more workgroups per compute unit), also
    // with streaming loads
    uint32_t rr[FIRST ? kRItems : 1], loc[kRItems];
    const uint64_t lt = lanemask_lt();
    // record idx of a slab (row r) is entry idx + row_off[r]
    auto slab_entry = [&](int64_t idx, int64_t r) -> int64_t { return idx + sl.row_off[r]; };
    // all of the segment's keys in flight at once, then the ranking
    // (a slab's values are loaded with their keys, so that each record's
    // entry is found once)
    V vpre[SRC == kSrcSlab && VB != 0 ? kRItems : 1];
    if constexpr (SRC == kSrcSlab) {
#pragma unroll
        for (int k = 0; k < kRItems; ++k) {
            const int64_t idx = segbase + int64_t(k) * kWave + lane;
            const int64_t r = idx < n ? int64_t(reinterpret_cast<const uint32_t*>(ex)[idx - base]) : 0;
            rr[k] = uint32_t(r);
            const int64_t e = slab_entry(idx, r);
            kr[k] = idx < n ? uint32_t(int64_t(sl.ci[e]) - sl.c0) : 0u;
            if constexpr (VB != 0) vpre[k] = idx < n ? static_cast<const V*>(sl.val)[e] : V(0);
        }
    }
#pragma unroll
    for (int k = 0; k < kRItems; ++k) {
        const int64_t idx = segbase + int64_t(k) * kWave + lane;
        const bool valid = idx < n;
        const uint32_t key = kr[k];
        const uint32_t d = (key >> shift) & mask;
        uint64_t peers = __ballot(valid);
#pragma unroll
        for (int b = 0; b < kRBits; ++b) {
            const bool bit = (d >> b) & 1u;
            const uint64_t bal = __ballot(bit);
            peers &= bit ? bal : ~bal;
        }
        uint32_t cur = 0;
        if (valid) cur = wcnt[w][d];
        const uint32_t rank = __popcll(peers & lt);
        loc[k] = cur + rank;
        if (valid && rank == 0) wcnt[w][d] = cur + uint32_t(__popcll(peers));
        if constexpr (SRC == kSrcCsr) {
            uint32_t field = 0;
            if (valid) {
                int64_t r, len;
                if (rstaged) {
                    const int64_t rl = reinterpret_cast<const uint32_t*>(ex)[idx - base];
                    r = rlo + rl;
                    len = rwin[rl + 1] - rwin[rl];
                } else {
                    r = last_leq_i64(rp, rlo, rhi, idx);
                    len = rp[r + 1] - rp[r];
                }
                field = uint32_t(r);
                if (lenbits > 0) {
                    const int64_t lmax = (int64_t(1) << lenbits) - 1;
                    field |= uint32_t(len < lmax ? len : lmax) << rowbits;
                }
            }
            rr[k] = field;
        }
    }
    __syncthreads();
    {
        const int d = threadIdx.x;
        uint32_t c[kWavesPerBlock];
        uint32_t tot = 0;
#pragma unroll
        for (int q = 0; q < kWavesPerBlock; ++q) {
            c[q] = wcnt[q][d];
            tot += c[q];
        }
        uint32_t all;
        uint32_t off = block_exclusive_scan(tot, wt, &all);
        gofs[d] = int64_t(offs[int64_t(d) * ntiles + tile]) - int64_t(off);
#pragma unroll
        for (int q = 0; q < kWavesPerBlock; ++q) {
            wcnt[q][d] = off;
            off += c[q];
        }
    }
    __syncthreads();
    // tile positions of the records (registers), then keys, rows and values in turn
#pragma unroll
    for (int k = 0; k < kRItems; ++k) {
        const int64_t idx = segbase + int64_t(k) * kWave + lane;
        if (idx < n) {
            const uint32_t d = (kr[k] >> shift) & mask;
            loc[k] += wcnt[w][d];
            ex[loc[k]] = V(kr[k]);
            dig[loc[k]] = uint8_t(d);
            if constexpr (OUT == kOutPlace) kslot[loc[k]] = uint16_t(kr[k]);
        }
    }
    __syncthreads();
    const int tile_n = int(min(int64_t(kRTile), n - base));
    for (int i = threadIdx.x; i < tile_n; i += kBlock) key_out[gofs[dig[i]] + i] = uint32_t(ex[i]);
    __syncthreads();
    if constexpr (FIRST) {
#pragma unroll
        for (int k = 0; k < kRItems; ++k)
            if (segbase + int64_t(k) * kWave + lane < n) ex[loc[k]] = V(rr[k]);
    } else {
        uint32_t rv[kRItems];
#pragma unroll
        for (int k = 0; k < kRItems; ++k) {
            const int64_t idx = segbase + int64_t(k) * kWave + lane;
            rv[k] = idx < n ? __builtin_nontemporal_load(row_in + idx) : 0u;
        }
#pragma unroll
        for (int k = 0; k < kRItems; ++k)
            if (segbase + int64_t(k) * kWave + lane < n) ex[loc[k]] = V(rv[k]);
    }
    __syncthreads();
    // full-row position of the record in slot i (kOutPlace)
    auto place = [&](int i) -> int64_t {
        const int64_t q = gofs[dig[i]] + i;
        return sl.before + q + sl.rp[sl.c0 + int64_t(kslot[i]) + 1];
    };
    for (int i = threadIdx.x; i < tile_n; i += kBlock) {
        if constexpr (OUT == kOutPlace)
            sl.f_ci[place(i)] = int32_t(ex[i]);
        else
            row_out[gofs[dig[i]] + i] = uint32_t(ex[i]);
    }
    if constexpr (VB != 0) {
        V vv[kRItems];
#pragma unroll
        for (int k = 0; k < kRItems; ++k) {
            const int64_t idx = segbase + int64_t(k) * kWave + lane;
            if constexpr (SRC == kSrcCsr)  // the entry index, or with val_in the entry's value
                vv[k] = val_in ? (idx < n ? __builtin_nontemporal_load(val_in + idx) : V(0)) : V(idx);
            else if constexpr (SRC == kSrcSlab)
                vv[k] = vpre[k];
            else
                vv[k] = idx < n ? __builtin_nontemporal_load(val_in + idx) : V(0);
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < kRItems; ++k)
            if (segbase + int64_t(k) * kWave + lane < n) ex[loc[k]] = vv[k];
        __syncthreads();
        for (int i = threadIdx.x; i < tile_n; i += kBlock) {
            if constexpr (OUT == kOutPlace)
                static_cast<V*>(sl.f_val)[place(i)] = ex[i];
            else
                val_out[gofs[dig[i]] + i] = ex[i];
        }
    }
}

// ---- local sort of the low key bits inside groups of equal high bits
//
// After stable passes over the high bits [L, nbits) the records of every
// value v of the high bits form one contiguous group, in input order.  One
// workgroup per v sorts its group stably by the low L <= kLBits bits: in LDS
// (the low bits and the records' indices in the group, 6-bit digits), then
// gathers the records into place; a group too large for LDS is sorted by the
// same workgroup over global memory, tile by tile.

constexpr int kLBits = 12;       // low bits sorted locally
constexpr int kLCap = 4096;      // records of a group sorted in LDS
constexpr int kLCapS = 2048;     // the same in the packed sort's first launch (half the LDS and registers)
constexpr int kLDig = 6;         // bits per local digit
constexpr uint32_t kNoGroup = 0xffffffffu;

// first and end position of every group of equal high bits (groups that do
// not occur keep kNoGroup); big, if given, is emptied as in digit_starts
// (eight keys per thread, read with 16-byte loads when the keys are aligned)
__global__ __launch_bounds__(kBlock) void group_bounds(const uint32_t* __restrict__ key, int64_t n, int L,
                                                       uint32_t* __restrict__ gstart, uint32_t* __restrict__ gend,
                                                       uint32_t* __restrict__ big) {
    if (big && blockIdx.x == 0 && threadIdx.x == 0) big[0] = 0;
    const int64_t p0 = (int64_t(blockIdx.x) * kBlock + threadIdx.x) * 8;
    if (p0 >= n) return;
    uint32_t k[9];  // key p0 - 1 (or none), then keys p0 .. p0 + 7
    k[0] = p0 > 0 ? key[p0 - 1] : 0u;
    if (p0 + 8 <= n && (reinterpret_cast<uintptr_t>(key + p0) & 15) == 0) {
        const uint4 a = reinterpret_cast<const uint4*>(key + p0)[0];
        const uint4 b = reinterpret_cast<const uint4*>(key + p0)[1];
        k[1] = a.x;
        k[2] = a.y;
        k[3] = a.z;
        k[4] = a.w;
        k[5] = b.x;
        k[6] = b.y;
        k[7] = b.z;
        k[8] = b.w;
    } else {
#pragma unroll
        for (int u = 0; u < 8; ++u) k[u + 1] = p0 + u < n ? key[p0 + u] : 0u;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int64_t p = p0 + u;
        if (p >= n) break;
        const uint32_t v = k[u + 1] >> L;
        if (p == 0 || (k[u] >> L) != v) {
            gstart[v] = uint32_t(p);
            if (p > 0) gend[k[u] >> L] = uint32_t(p);
        }
        if (p == n - 1) gend[v] = uint32_t(n);
    }
}

// Group starts from the passes' scanned histograms, without reading the
// sorted keys, when the high bits take one or two passes.  With one pass
// (digit d of w1 bits) group d starts where the pass put the digit's first
// record.  With two (d1 of w1 bits, then d2), the groups are (d2, d1) in that
// order, and the records of (d2, d1) come from the second pass's input tiles
// in order: those before the tile t1 holding the first record of d1 (all of
// smaller d1), then those of t1 before that record.  So group (d2, d1) starts
// at the second pass's position of t1's first d2 record, plus the d2 records
// of t1 before d1 begins.  gstart gets 2^h + 1 entries (the last is n): group
// g occupies [gstart[g], gstart[g + 1]).

// first1[d] = position of the first record of digit d after the first pass
// (hist: the first pass's scanned histogram, digit-major)
// (big, if given: the packed sort's list of large groups, emptied here)
__global__ __launch_bounds__(kBlock) void digit_starts(const uint32_t* __restrict__ hist, int64_t ntiles, int ndig,
                                                       uint32_t* __restrict__ first1, int64_t n,
                                                       uint32_t* __restrict__ big) {
    const int d = threadIdx.x;
    if (d < ndig) first1[d] = hist[int64_t(d) * ntiles];
    if (d == 0) {
        first1[ndig] = uint32_t(n);
        if (big) big[0] = 0;
    }
}

// one workgroup per d1: the d2 counts of tile t1 before first1[d1] (keys:
// the first pass's output), then the starts of groups (d2, d1) for every d2
// (hist: the second pass's scanned histogram)
__global__ __launch_bounds__(kBlock) void group_starts(const uint32_t* __restrict__ key, int64_t n, int L, int w1,
                                                       int w2, const uint32_t* __restrict__ first1,
                                                       const uint32_t* __restrict__ hist, int64_t ntiles,
                                                       uint32_t* __restrict__ gstart) {
    __shared__ uint32_t cnt[kDigits];
    const uint32_t d1 = blockIdx.x;
    const int nd2 = 1 << w2;
    cnt[threadIdx.x] = 0;
    __syncthreads();
    const int64_t f = first1[d1];
    const int64_t t1 = f / kRTile;
    const uint32_t m2 = uint32_t(nd2 - 1);
    if (t1 < ntiles)
        for (int64_t p = t1 * kRTile + threadIdx.x; p < f; p += kBlock) atomicAdd(&cnt[(key[p] >> (L + w1)) & m2], 1u);
    __syncthreads();
    const int d2 = threadIdx.x;
    if (d2 < nd2) {
        uint32_t st;
        if (t1 < ntiles)
            st = hist[int64_t(d2) * ntiles + t1] + cnt[d2];
        else  // d1 empty at the end: every group (d2, d1) starts where d2's records end
            st = d2 + 1 < nd2 ? hist[int64_t(d2 + 1) * ntiles] : uint32_t(n);
        gstart[(uint32_t(d2) << w1) | d1] = st;
    }
    if (d1 == 0 && threadIdx.x == 0) gstart[uint32_t(1) << (w1 + w2)] = uint32_t(n);
}

// one stable pass of the LDS sort: (dig, idx) of S <= kLCap records by bits
// [sh, sh + w) of dig, from the *_in arrays to the *_out arrays
template <int CAP>
__device__ inline void lds_pass(const uint16_t* dig_in, const uint16_t* idx_in, uint16_t* dig_out, uint16_t* idx_out,
                                int S, int sh, int w, uint32_t (*wcnt)[1 << kLDig], uint32_t* wt) {
    constexpr int kCh = CAP / kWavesPerBlock / kWave;  // chunks of a wave's segment
    const int wv = threadIdx.x / kWave;
    const int lane = lane_id();
    const uint32_t m = (1u << w) - 1u;
    const int seg = ((S + kWavesPerBlock - 1) / kWavesPerBlock + kWave - 1) / kWave * kWave;
    const int s0 = wv * seg, s1 = min(S, s0 + seg);
    wcnt[wv][lane] = 0;
    __syncthreads();
    const uint64_t lt = lanemask_lt();
    const int nch = seg / kWave;  // (the same in every wavefront)
    uint32_t loc[kCh];
    uint32_t dd[kCh];
#pragma unroll
    for (int c = 0; c < kCh; ++c) {
        if (c >= nch) break;
        const int i = s0 + c * kWave + lane;
        const bool valid = i < s1;
        const uint32_t d = valid ? (uint32_t(dig_in[i]) >> sh) & m : 0u;
        uint64_t peers = __ballot(valid);
        for (int b = 0; b < w; ++b) {
            const bool bit = (d >> b) & 1u;
            const uint64_t bal = __ballot(bit);
            peers &= bit ? bal : ~bal;
        }
        uint32_t cur = 0;
        if (valid) cur = wcnt[wv][d];
        const uint32_t rank = __popcll(peers & lt);
        loc[c] = cur + rank;
        dd[c] = d;
        if (valid && rank == 0) wcnt[wv][d] = cur + uint32_t(__popcll(peers));
    }
    __syncthreads();
    {
        // exclusive offsets in (digit, wavefront) order: thread t = digit * waves + wave
        const int d = threadIdx.x / kWavesPerBlock, q = threadIdx.x % kWavesPerBlock;
        const uint32_t v = wcnt[q][d];
        uint32_t tot;
        const uint32_t off = block_exclusive_scan(v, wt, &tot);
        __syncthreads();
        wcnt[q][d] = off;
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < kCh; ++c) {
        if (c >= nch) break;
        const int i = s0 + c * kWave + lane;
        if (i < s1) {
            const uint32_t dest = wcnt[wv][dd[c]] + loc[c];
            dig_out[dest] = dig_in[i];
            idx_out[dest] = idx_in[i];
        }
    }
    __syncthreads();
}

// one stable pass of the global-memory sort of a large group [b0, b0 + S):
// by bits [sh, sh + w) of the key, from the *i arrays to the *o arrays, in
// tiles of kBlock records in order
template <typename E>
__device__ inline void group_pass(const uint32_t* ki, const uint32_t* ri, const E* ei, uint32_t* ko, uint32_t* ro,
                                  E* eo, int64_t b0, int64_t S, int sh, int w, uint32_t* base,
                                  uint32_t (*wcnt)[1 << kLDig], uint32_t* wt) {
    const int wv = threadIdx.x / kWave;
    const int lane = lane_id();
    const uint32_t m = (1u << w) - 1u;
    if (threadIdx.x < (1 << kLDig)) base[threadIdx.x] = 0;
    __syncthreads();
    for (int64_t i = threadIdx.x; i < S; i += kBlock) atomicAdd(&base[(ki[b0 + i] >> sh) & m], 1u);
    __syncthreads();
    {
        const uint32_t v = threadIdx.x < (1 << kLDig) ? base[threadIdx.x] : 0u;
        uint32_t tot;
        const uint32_t off = block_exclusive_scan(v, wt, &tot);
        __syncthreads();
        if (threadIdx.x < (1 << kLDig)) base[threadIdx.x] = off;
    }
    __syncthreads();
    const uint64_t lt = lanemask_lt();
    for (int64_t t0 = 0; t0 < S; t0 += kBlock) {
        const int64_t i = t0 + threadIdx.x;
        const bool valid = i < S;
        const uint32_t kv = valid ? ki[b0 + i] : 0u;
        const uint32_t d = (kv >> sh) & m;
        uint64_t peers = __ballot(valid);
        for (int b = 0; b < w; ++b) {
            const bool bit = (d >> b) & 1u;
            const uint64_t bal = __ballot(bit);
            peers &= bit ? bal : ~bal;
        }
        const uint32_t rank = __popcll(peers & lt);
        wcnt[wv][lane] = 0;
        __syncthreads();
        if (valid && rank == 0) wcnt[wv][d] = uint32_t(__popcll(peers));
        __syncthreads();
        uint32_t before = 0;
        for (int q = 0; q < wv; ++q) before += wcnt[q][d];
        if (valid) {
            const int64_t dest = b0 + int64_t(base[d] + before + rank);
            ko[dest] = kv;
            ro[dest] = ri[b0 + i];
            eo[dest] = ei[b0 + i];
        }
        __syncthreads();
        if (threadIdx.x < (1 << kLDig)) {
            uint32_t add = 0;
            for (int q = 0; q < kWavesPerBlock; ++q) add += wcnt[q][threadIdx.x];
            base[threadIdx.x] += add;
        }
        __syncthreads();
    }
}

// Group v = blockIdx.x: sort [gstart[v], gend[v]) of (kx, rx, ex) stably by
// the low L bits of the key into (ky, ry, ey).  A group over kLCap records
// uses x and y in turn over global memory and ends in y.
__global__ __launch_bounds__(kBlock) void local_sort(uint32_t* __restrict__ kx, uint32_t* __restrict__ rx,
                                                     uint32_t* __restrict__ ex, uint32_t* __restrict__ ky,
                                                     uint32_t* __restrict__ ry, uint32_t* __restrict__ ey,
                                                     const uint32_t* __restrict__ gstart,
                                                     const uint32_t* __restrict__ gend, int L) {
    __shared__ uint16_t dg[2][kLCap];
    __shared__ uint16_t ix[2][kLCap];
    __shared__ uint32_t wcnt[kWavesPerBlock][1 << kLDig];
    __shared__ uint32_t base[1 << kLDig];
    __shared__ uint32_t wt[kWavesPerBlock];
    static_assert(kWavesPerBlock * (1 << kLDig) == kBlock, "one thread per (digit, wavefront)");
    static_assert(kLCap <= 65536, "indices in a group are 16 bits");
    const uint32_t g0 = gstart[blockIdx.x];
    if (g0 == kNoGroup) return;
    const int64_t b0 = g0;
    const int64_t S = int64_t(gend[blockIdx.x]) - b0;
    if (S <= 0) return;  // (an empty group, when the starts come from the histograms)
    const uint32_t lmask = (1u << L) - 1u;
    if (S <= kLCap) {
        for (int i = threadIdx.x; i < S; i += kBlock) {
            dg[0][i] = uint16_t(kx[b0 + i] & lmask);
            ix[0][i] = uint16_t(i);
        }
        __syncthreads();
        int cur = 0;
        for (int sh = 0; sh < L; sh += kLDig) {
            lds_pass<kLCap>(dg[cur], ix[cur], dg[cur ^ 1], ix[cur ^ 1], int(S), sh, min(kLDig, L - sh), wcnt, wt);
            cur ^= 1;
        }
        for (int j = threadIdx.x; j < S; j += kBlock) {
            const int64_t src = b0 + ix[cur][j];
            ky[b0 + j] = kx[src];
            ry[b0 + j] = rx[src];
            ey[b0 + j] = ex[src];
        }
        return;
    }
    // a large group: passes over global memory, x -> y -> x ..., ending in y
    int npass = 0;
    for (int sh = 0; sh < L; sh += kLDig) {
        const bool to_y = (npass & 1) == 0;
        group_pass(to_y ? kx : ky, to_y ? rx : ry, to_y ? ex : ey, to_y ? ky : kx, to_y ? ry : rx, to_y ? ey : ex, b0,
                   S, sh, min(kLDig, L - sh), base, wcnt, wt);
        ++npass;
    }
    if ((npass & 1) == 0) {
        for (int64_t i = threadIdx.x; i < S; i += kBlock) {
            ky[b0 + i] = kx[b0 + i];
            ry[b0 + i] = rx[b0 + i];
            ey[b0 + i] = ex[b0 + i];
        }
    }
}

// ---- the column index in partner-run form, straight from the local sort
//
// Instead of a sorted copy of the records, the workgroup of a group writes
// the key (the row) and value of every entry at its sorted position, and in
// lower mode every entry's partner run {first position of its column, its
// own position}: the entries of its column with a smaller row.  (The last
// entry of a column is never a partner; its slot is written but not read.)

template <int VB>
__device__ inline typename ValT<VB>::T entry_value(const LocalPack& pk, uint32_t ent) {
    if constexpr (VB == 0)
        return 0;
    else
        return static_cast<const typename ValT<VB>::T*>(pk.vals_b)[ent];
}

// v: the entry's value (VB 4 or 8), read by the caller; last: the entry ends
// column col
template <int VB, bool JAC>
__device__ inline void emit_entry(const LocalPack& pk, int64_t pos, uint32_t field, uint32_t ent, int64_t cstart,
                                  typename ValT<VB>::T v, bool last, uint32_t col) {
    if (pk.ccount && last) pk.ccount[col] = uint32_t(pos - cstart + 1);
    if (pk.vsrc) nt_store(ent, pk.vsrc + pos);
    const uint32_t rowmask = pk.rowbits >= 32 ? 0xffffffffu : ((1u << pk.rowbits) - 1u);
    const uint32_t row = field & rowmask;
    if constexpr (JAC) {
        if (!pk.val) {
            nt_store(field, pk.key + pos);  // the row and its saturated length
        } else {
            nt_store(row, pk.key + pos);
            const uint32_t lmax = pk.lenbits > 0 ? (1u << pk.lenbits) - 1u : 0u;
            const uint32_t lf = pk.lenbits > 0 ? field >> pk.rowbits : lmax;
            nt_store(lf < lmax ? int32_t(lf) : int32_t(pk.rp_b[row + 1] - pk.rp_b[row]),
                     static_cast<int32_t*>(pk.val) + pos);
        }
    } else {
        nt_store(row, pk.key + pos);
        if constexpr (VB != 0) nt_store(v, static_cast<typename ValT<VB>::T*>(pk.val) + pos);
    }
    if (pk.run && pos > cstart) set_run(pk.run, ent, uint32_t(cstart), uint32_t(pos));
}

// The third field of the records: the entry index, or with CARRY the
// entry's value itself (VB bytes, carried through the passes).
template <int VB, bool CARRY>
using EntT = typename std::conditional<CARRY, typename ValT<VB>::T, uint32_t>::type;

// The LDS path of local_sort_pack: the group of S <= CAP records at b0.
// Returns the number of distinct columns (the same in every thread).
template <int VB, bool JAC, int CAP, bool CARRY>
__device__ inline uint32_t pack_group_lds(const uint32_t* __restrict__ kx, const uint32_t* __restrict__ rx,
                                          const EntT<VB, CARRY>* __restrict__ ex, int64_t b0, int S, int L,
                                          const LocalPack& pk, uint16_t (*dg)[CAP], uint16_t (*ix)[CAP],
                                          uint32_t (*wcnt)[1 << kLDig], uint32_t* wt) {
    static_assert(CAP % kBlock == 0 && CAP <= 65536, "whole rounds of the workgroup; 16-bit indices");
    constexpr int kPer = CAP / kBlock;
    const uint32_t lmask = (1u << L) - 1u;
    // every global access of the group is issued as one batch per thread
    // (kPer records, unrolled), so a workgroup waits on memory a few times
    // rather than once per record stride
    {
        uint32_t kv[kPer];
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int i = threadIdx.x + k * kBlock;
            kv[k] = i < S ? kx[b0 + i] : 0u;
        }
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int i = threadIdx.x + k * kBlock;
            if (i < S) {
                dg[0][i] = uint16_t(kv[k] & lmask);
                ix[0][i] = uint16_t(i);
            }
        }
    }
    __syncthreads();
    int cur = 0;
    for (int sh = 0; sh < L; sh += kLDig) {
        lds_pass<CAP>(dg[cur], ix[cur], dg[cur ^ 1], ix[cur ^ 1], S, sh, min(kLDig, L - sh), wcnt, wt);
        cur ^= 1;
    }
    // row fields and entry indices (or values) in sorted order (in flight
    // during the scan below)
    uint32_t rv[kPer];
    EntT<VB, CARRY> ev[kPer];
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
        const int j = threadIdx.x + k * kBlock;
        if (j < S) {
            const int64_t src = b0 + ix[cur][j];
            rv[k] = rx[src];
            ev[k] = ex[src];
        }
    }
    // first position of every entry's column: the positions where the low
    // bits change, then a max-scan (kPer consecutive positions per thread)
    uint16_t* cs = dg[cur ^ 1];
    uint32_t distinct;
    {
        const int j0 = threadIdx.x * kPer;
        uint32_t run[kPer];
        uint32_t mx = 0, nst = 0;
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int j = j0 + k;
            if (j < S && (j == 0 || dg[cur][j - 1] != dg[cur][j])) {
                mx = uint32_t(j);
                ++nst;
            }
            run[k] = mx;
        }
        uint32_t all;
        const uint32_t before = block_exclusive_max(mx, wt, &all);
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int j = j0 + k;
            if (j < S) cs[j] = uint16_t(max(run[k], before));
        }
        (void)block_exclusive_scan(nst, wt, &distinct);
    }
    __syncthreads();
    typename ValT<VB>::T vv[kPer];
#pragma unroll
    for (int k = 0; k < kPer; ++k)
        if (threadIdx.x + k * kBlock < S) {
            if constexpr (CARRY)
                vv[k] = ev[k];
            else
                vv[k] = entry_value<VB>(pk, ev[k]);
        }
    const uint32_t hi = kx[b0] & ~lmask;  // the group's high column bits
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
        const int j = threadIdx.x + k * kBlock;
        if (j < S) {
            const uint32_t lo = dg[cur][j];
            const bool last = j == S - 1 || dg[cur][j + 1] != lo;
            const uint32_t ent = CARRY ? 0u : uint32_t(ev[k]);  // (with CARRY no entry index is written)
            emit_entry<VB, JAC>(pk, b0 + j, rv[k], ent, b0 + cs[j], vv[k], last, hi | lo);
        }
    }
    return distinct;
}

// The same for a group of any size, by passes over global memory (x -> y ->
// x ..., ending in y), then the output a tile at a time.
template <int VB, bool JAC, bool CARRY>
__device__ inline uint32_t pack_group_global(uint32_t* __restrict__ kx, uint32_t* __restrict__ rx,
                                             EntT<VB, CARRY>* __restrict__ ex, uint32_t* __restrict__ ky,
                                             uint32_t* __restrict__ ry, EntT<VB, CARRY>* __restrict__ ey, int64_t b0,
                                             int64_t S, int L, const LocalPack& pk, uint32_t* base,
                                             uint32_t (*wcnt)[1 << kLDig], uint32_t* wt) {
    int npass = 0;
    for (int sh = 0; sh < L; sh += kLDig) {
        const bool to_y = (npass & 1) == 0;
        group_pass(to_y ? kx : ky, to_y ? rx : ry, to_y ? ex : ey, to_y ? ky : kx, to_y ? ry : rx, to_y ? ey : ex, b0,
                   S, sh, min(kLDig, L - sh), base, wcnt, wt);
        ++npass;
    }
    const uint32_t* ks = (npass & 1) ? ky : kx;
    const uint32_t* rs = (npass & 1) ? ry : rx;
    const EntT<VB, CARRY>* es = (npass & 1) ? ey : ex;
    // the column start carried over from tile to tile
    uint32_t carry = 0, distinct = 0;
    for (int64_t t0 = 0; t0 < S; t0 += kBlock) {
        const int64_t j = t0 + threadIdx.x;
        const bool st = j < S && (j == 0 || ks[b0 + j - 1] != ks[b0 + j]);
        const uint32_t v = st ? uint32_t(j) : 0u;
        uint32_t all;
        const uint32_t cstart = max(max(block_exclusive_max(v, wt, &all), v), carry);
        uint32_t tot;
        (void)block_exclusive_scan(st ? 1u : 0u, wt, &tot);
        distinct += tot;
        if (j < S) {
            const uint32_t col = ks[b0 + j];
            const bool last = j == S - 1 || ks[b0 + j + 1] != col;
            typename ValT<VB>::T v;
            uint32_t ent = 0;
            if constexpr (CARRY) {
                v = es[b0 + j];
            } else {
                ent = es[b0 + j];
                v = entry_value<VB>(pk, ent);
            }
            emit_entry<VB, JAC>(pk, b0 + j, rs[b0 + j], ent, b0 + cstart, v, last, col);
        }
        carry = max(carry, all);
    }
    return distinct;
}

__device__ inline void add_kept(const LocalPack& pk, int64_t S, uint32_t distinct) {
    if (threadIdx.x == 0 && pk.kept)
        atomicAdd(reinterpret_cast<unsigned long long*>(pk.kept),
                  (unsigned long long)(pk.drop_last ? S - int64_t(distinct) : S));
}

// Group v = blockIdx.x, of S <= kLCapS records: sorted in LDS and written
// as the column index.  A larger group is appended to the list big (big[0]
// its length, zero on entry; then the group numbers) for
// local_sort_pack_big.  The small capacity halves the LDS and the registers
// of a workgroup, which doubles the workgroups a compute unit holds.
template <int VB, bool JAC, bool CARRY>
__global__ __launch_bounds__(kBlock) void local_sort_pack(const uint32_t* __restrict__ kx,
                                                          const uint32_t* __restrict__ rx,
                                                          const EntT<VB, CARRY>* __restrict__ ex,
                                                          const uint32_t* __restrict__ gstart,
                                                          const uint32_t* __restrict__ gend, int L, LocalPack pk,
                                                          uint32_t* __restrict__ big) {
    __shared__ uint16_t dg[2][kLCapS];
    __shared__ uint16_t ix[2][kLCapS];
    __shared__ uint32_t wcnt[kWavesPerBlock][1 << kLDig];
    __shared__ uint32_t wt[kWavesPerBlock];
    const uint32_t g0 = gstart[blockIdx.x];
    if (g0 == kNoGroup) return;
    const int64_t b0 = g0;
    const int64_t S = int64_t(gend[blockIdx.x]) - b0;
    if (S <= 0) return;  // (an empty group, when the starts come from the histograms)
    if (S > kLCapS) {
        if (threadIdx.x == 0) big[1 + atomicAdd(big, 1u)] = blockIdx.x;
        return;
    }
    add_kept(pk, S, pack_group_lds<VB, JAC, kLCapS, CARRY>(kx, rx, ex, b0, int(S), L, pk, dg, ix, wcnt, wt));
}

// The groups local_sort_pack listed, shared out over the grid: in LDS up to
// kLCap records, over global memory (x and y in turn) beyond.
template <int VB, bool JAC, bool CARRY>
__global__ __launch_bounds__(kBlock) void local_sort_pack_big(uint32_t* __restrict__ kx, uint32_t* __restrict__ rx,
                                                              EntT<VB, CARRY>* __restrict__ ex,
                                                              uint32_t* __restrict__ ky, uint32_t* __restrict__ ry,
                                                              EntT<VB, CARRY>* __restrict__ ey,
                                                              const uint32_t* __restrict__ gstart,
                                                              const uint32_t* __restrict__ gend, int L,
                                                              LocalPack pk, const uint32_t* __restrict__ big) {
    __shared__ uint16_t dg[2][kLCap];
    __shared__ uint16_t ix[2][kLCap];
    __shared__ uint32_t wcnt[kWavesPerBlock][1 << kLDig];
    __shared__ uint32_t base[1 << kLDig];
    __shared__ uint32_t wt[kWavesPerBlock];
    const uint32_t nbig = big[0];
    for (uint32_t q = blockIdx.x; q < nbig; q += gridDim.x) {
        const uint32_t g = big[1 + q];
        const int64_t b0 = gstart[g];
        const int64_t S = int64_t(gend[g]) - b0;
        const uint32_t distinct =
            S <= kLCap ? pack_group_lds<VB, JAC, kLCap, CARRY>(kx, rx, ex, b0, int(S), L, pk, dg, ix, wcnt, wt)
                       : pack_group_global<VB, JAC, CARRY>(kx, rx, ex, ky, ry, ey, b0, S, L, pk, base, wcnt, wt);
        add_kept(pk, S, distinct);
        __syncthreads();  // (the shared arrays serve the next group)
    }
}

template <int VB, int SRC = kSrcArrays, int OUT = kOutArrays>
void run_pass(const uint32_t* ki, const uint32_t* ri, const void* vi, uint32_t* ko, uint32_t* ro, void* vo, int64_t n,
              int shift, uint32_t mask, uint32_t* hist, void* scan_tmp, hipStream_t s, const int64_t* rp = nullptr,
              int64_t m = 0, const int64_t* trow = nullptr, int rowbits = 0, int lenbits = 0,
              const SlabIo& sl = SlabIo(), bool counted = false) {
    using V = typename ValT<VB>::T;
    const int64_t ntiles = (n + kRTile - 1) / kRTile;
    const unsigned grid = unsigned((ntiles + kXcds - 1) / kXcds * kXcds);
    if constexpr (SRC == kSrcSlab)
        radix_hist_slab<<<dim3(grid), dim3(kBlock), 0, s>>>(n, mask, hist, ntiles, rp, m, trow, sl);
    else if (!counted)
        radix_hist<<<dim3(grid), dim3(kBlock), 0, s>>>(ki, n, shift, mask, hist, ntiles);
    scan_u32(hist, hist, ntiles * kDigits, nullptr, scan_tmp, s);
    radix_scatter<VB, SRC, OUT><<<dim3(unsigned((ntiles + kXcds - 1) / kXcds * kXcds)), dim3(kBlock), 0, s>>>(
        ki, ri, static_cast<const V*>(vi), ko, ro, static_cast<V*>(vo), n, shift, mask, hist, ntiles, rp, m, trow, rowbits,
        lenbits, sl);
}

// Digit widths of the passes for an nbits-bit key: as few passes as 8-bit
// digits need, the bits spread evenly over them (narrower digits give each
// tile longer runs per digit, so fuller lines are written).  Returns the
// number of passes (at least one).
int digit_plan(int nbits, int (&width)[8]) {
    const int passes = nbits > 0 ? (nbits + kRBits - 1) / kRBits : 1;
    const int base = nbits / passes, extra = nbits % passes;
    for (int i = 0; i < passes; ++i) width[i] = base + (i < extra ? 1 : 0);
    return passes;
}

}  // namespace

// Local-sort plan of a CSR column sort: the high h = nbits - L bits by passes,
// the low L (1..kLBits) bits inside groups of equal high bits, about 2048
// records per group on average.  Used for wide keys over many entries
// (SPSYRK_LOCAL_SORT=1 forces it wherever it applies, =0 turns it off; read
// at every call).  Returns L, or 0 for passes over all bits.
int local_bits(int64_t n, int nbits) {
    const char* e = std::getenv("SPSYRK_LOCAL_SORT");
    const bool force = e && e[0] == '1';
    if (e && e[0] == '0') return 0;
    if (!force && (nbits < 22 || n < (int64_t(1) << 20))) return 0;
    int h = nbits - kLBits;
    const int hg = bit_width_u64(uint64_t(n / 2048));  // groups of about 2048 records
    if (hg > h) h = hg;
    if (h < 1) h = 1;
    const int L = nbits - h;
    return L >= 1 ? L : 0;
}

void radix_first_digit(int64_t n, int nbits, int* shift, uint32_t* mask) {
    const int L = local_bits(n, nbits);
    int width[8];
    digit_plan(nbits - L, width);
    *shift = L;
    *mask = (1u << width[0]) - 1u;
}

size_t radix_csr_tmp_bytes(int64_t n, int nbits) {
    const int L = local_bits(n, nbits);
    const size_t groups = L ? (size_t(1) << (nbits - L)) : 0;
    // group starts (groups + 1), ends and the list of large groups (length,
    // then up to groups entries), then the first pass's digit starts
    return radix_tmp_bytes(n) + 3 * (((groups + 1) * sizeof(uint32_t) + 255) & ~size_t(255)) +
           ((size_t(kDigits + 1) * sizeof(uint32_t) + 255) & ~size_t(255));
}

size_t radix_tmp_bytes(int64_t n) {
    const int64_t ntiles = (n + kRTile - 1) / kRTile;
    const size_t hist = size_t(ntiles) * kDigits * sizeof(uint32_t);
    const size_t table = size_t(ntiles + 1) * sizeof(int64_t);
    return ((hist + 255) & ~size_t(255)) + ((table + 255) & ~size_t(255)) + scan_tmp_bytes(ntiles * kDigits);
}

int radix_sort_csr(const int32_t* col_idx, const int64_t* rp, int64_t m, int rowbits, int lenbits, uint32_t* key_a,
                   uint32_t* key_b, uint32_t* row_a, uint32_t* row_b, uint32_t* ent_a, uint32_t* ent_b, int64_t n,
                   int nbits, void* tmp, hipStream_t s, const LocalPack* pk, uint32_t* hist1,
                   const int64_t* trow1) {
    if (n <= 0) return 0;
    const int64_t ntiles = (n + kRTile - 1) / kRTile;
    uint32_t* hist = static_cast<uint32_t*>(tmp);
    const size_t hist_bytes = (size_t(ntiles) * kDigits * sizeof(uint32_t) + 255) & ~size_t(255);
    const size_t table_bytes = (size_t(ntiles + 1) * sizeof(int64_t) + 255) & ~size_t(255);
    int64_t* trow = reinterpret_cast<int64_t*>(static_cast<char*>(tmp) + hist_bytes);
    void* scan_tmp = static_cast<char*>(tmp) + hist_bytes + table_bytes;
    // passes over all bits, or over the high bits followed by the local sort
    const int L = local_bits(n, nbits);
    int width[8];
    const int passes = digit_plan(nbits - L, width);
    // bytes of the values carried in place of the entry indices (local sort only)
    const int cv = pk && L ? pk->carried : 0;
    // first pass straight from the CSR arrays (into the b buffers), at least
    // one pass; the row of every tile's first entry comes from a table
    // with the local sort: the groups' starts (and ends), and the first
    // pass's digit starts
    const size_t groups = L ? size_t(1) << (nbits - L) : 0;
    uint32_t* gstart = nullptr;
    uint32_t* gend = nullptr;
    uint32_t* first1 = nullptr;
    uint32_t* big = nullptr;
    if (L) {
        const size_t gbytes = ((groups + 1) * sizeof(uint32_t) + 255) & ~size_t(255);
        gstart = reinterpret_cast<uint32_t*>(static_cast<char*>(tmp) + radix_tmp_bytes(n));
        gend = gstart + gbytes / sizeof(uint32_t);
        big = gend + gbytes / sizeof(uint32_t);
        first1 = big + gbytes / sizeof(uint32_t);
    }
    // group starts from the histograms when the high bits take one or two passes
    const bool from_hist = L && passes <= 2;
    int cur = 1;
    {
        PhaseTimer passes_timer(SPSYRK_PHASE_COLINDEX_PASSES, s);
        if (!trow1) tile_first_rows(rp, m, kRTile, trow, s);
        uint32_t* h1 = hist1 ? hist1 : hist;
        const uint32_t* ck = reinterpret_cast<const uint32_t*>(col_idx);
        const int64_t* tr = trow1 ? trow1 : trow;
        if (cv == 8)
            run_pass<8, kSrcCsr>(ck, nullptr, pk->vals_b, key_b, row_b, ent_b, n, L, (1u << width[0]) - 1u, h1,
                                 scan_tmp, s, rp, m, tr, rowbits, lenbits, SlabIo(), hist1 != nullptr);
        else
            run_pass<4, kSrcCsr>(ck, nullptr, cv == 4 ? pk->vals_b : nullptr, key_b, row_b, ent_b, n, L,
                                 (1u << width[0]) - 1u, h1, scan_tmp, s, rp, m, tr, rowbits, lenbits, SlabIo(),
                                 hist1 != nullptr);
        if (from_hist)
            digit_starts<<<1, kBlock, 0, s>>>(h1, ntiles, 1 << width[0], passes == 1 ? gstart : first1, n, big);
        int shift = L + width[0];
        for (int ps = 1; ps < passes; shift += width[ps], ++ps) {
            const uint32_t mask = (1u << width[ps]) - 1u;
            uint32_t* ki = cur ? key_b : key_a;
            uint32_t* ko = cur ? key_a : key_b;
            uint32_t* ri = cur ? row_b : row_a;
            uint32_t* ro = cur ? row_a : row_b;
            uint32_t* vi = cur ? ent_b : ent_a;
            uint32_t* vo = cur ? ent_a : ent_b;
            if (cv == 8)
                run_pass<8>(ki, ri, vi, ko, ro, vo, n, shift, mask, hist, scan_tmp, s);
            else
                run_pass<4>(ki, ri, vi, ko, ro, vo, n, shift, mask, hist, scan_tmp, s);
            cur ^= 1;
        }
        if (from_hist && passes == 2)
            group_starts<<<1u << width[0], kBlock, 0, s>>>(key_b, n, L, width[0], width[1], first1, hist, ntiles,
                                                           gstart);
    }
    if (L == 0) return cur;
    // groups of equal high bits, each sorted by the low L bits into the other buffers
    uint32_t* kx = cur ? key_b : key_a;
    uint32_t* rx = cur ? row_b : row_a;
    uint32_t* ex = cur ? ent_b : ent_a;
    if (from_hist) {
        gend = gstart + 1;  // group g ends where group g + 1 starts
    } else {
        fill_u32(gstart, int64_t(groups), kNoGroup, s);
        group_bounds<<<unsigned((n + 8 * kBlock - 1) / (8 * kBlock)), kBlock, 0, s>>>(kx, n, L, gstart, gend, big);
    }
    uint32_t* ky = cur ? key_a : key_b;
    uint32_t* ry = cur ? row_a : row_b;
    uint32_t* ey = cur ? ent_a : ent_b;
    if (pk) {
        const unsigned g = unsigned(groups);
        // the large groups (listed by the first launch) on a grid of at most
        // four workgroups per compute unit
        const unsigned gb = unsigned(std::min<size_t>(groups, 1024));
        PhaseTimer pack_timer(SPSYRK_PHASE_COLINDEX_PACK, s);
        if (pk->jac) {
            local_sort_pack<0, true, false><<<g, kBlock, 0, s>>>(kx, rx, ex, gstart, gend, L, *pk, big);
            local_sort_pack_big<0, true, false><<<gb, kBlock, 0, s>>>(kx, rx, ex, ky, ry, ey, gstart, gend, L, *pk,
                                                                      big);
        } else if (cv == 8) {
            using V = ValT<8>::T;
            V* vx = reinterpret_cast<V*>(ex);
            V* vy = reinterpret_cast<V*>(ey);
            local_sort_pack<8, false, true><<<g, kBlock, 0, s>>>(kx, rx, vx, gstart, gend, L, *pk, big);
            local_sort_pack_big<8, false, true><<<gb, kBlock, 0, s>>>(kx, rx, vx, ky, ry, vy, gstart, gend, L, *pk,
                                                                      big);
        } else if (cv == 4) {
            local_sort_pack<4, false, true><<<g, kBlock, 0, s>>>(kx, rx, ex, gstart, gend, L, *pk, big);
            local_sort_pack_big<4, false, true><<<gb, kBlock, 0, s>>>(kx, rx, ex, ky, ry, ey, gstart, gend, L, *pk,
                                                                      big);
        } else if (pk->vbytes == 8) {
            local_sort_pack<8, false, false><<<g, kBlock, 0, s>>>(kx, rx, ex, gstart, gend, L, *pk, big);
            local_sort_pack_big<8, false, false><<<gb, kBlock, 0, s>>>(kx, rx, ex, ky, ry, ey, gstart, gend, L, *pk,
                                                                       big);
        } else if (pk->vbytes == 4) {
            local_sort_pack<4, false, false><<<g, kBlock, 0, s>>>(kx, rx, ex, gstart, gend, L, *pk, big);
            local_sort_pack_big<4, false, false><<<gb, kBlock, 0, s>>>(kx, rx, ex, ky, ry, ey, gstart, gend, L, *pk,
                                                                       big);
        } else {
            local_sort_pack<0, false, false><<<g, kBlock, 0, s>>>(kx, rx, ex, gstart, gend, L, *pk, big);
            local_sort_pack_big<0, false, false><<<gb, kBlock, 0, s>>>(kx, rx, ex, ky, ry, ey, gstart, gend, L, *pk,
                                                                       big);
        }
        return -1;
    }
    local_sort<<<unsigned(groups), kBlock, 0, s>>>(kx, rx, ex, ky, ry, ey, gstart, gend, L);
    return cur ^ 1;
}

int radix_sort(uint32_t* key_a, uint32_t* key_b, uint32_t* row_a, uint32_t* row_b, void* val_a, void* val_b,
               int vbytes, int64_t n, int nbits, void* tmp, hipStream_t s) {
    if (n <= 1 || nbits <= 0) return 0;
    const int64_t ntiles = (n + kRTile - 1) / kRTile;
    uint32_t* hist = static_cast<uint32_t*>(tmp);
    const size_t hist_bytes = (size_t(ntiles) * kDigits * sizeof(uint32_t) + 255) & ~size_t(255);
    void* scan_tmp = static_cast<char*>(tmp) + hist_bytes;
    int width[8];
    const int passes = digit_plan(nbits, width);
    int cur = 0;
    int shift = 0;
    for (int ps = 0; ps < passes; shift += width[ps], ++ps) {
        const uint32_t mask = (1u << width[ps]) - 1u;
        uint32_t* ki = cur ? key_b : key_a;
        uint32_t* ko = cur ? key_a : key_b;
        uint32_t* ri = cur ? row_b : row_a;
        uint32_t* ro = cur ? row_a : row_b;
        void* vi = cur ? val_b : val_a;
        void* vo = cur ? val_a : val_b;
        if (vbytes == 8)
            run_pass<8>(ki, ri, vi, ko, ro, vo, n, shift, mask, hist, scan_tmp, s);
        else if (vbytes == 4)
            run_pass<4>(ki, ri, vi, ko, ro, vo, n, shift, mask, hist, scan_tmp, s);
        else
            run_pass<0>(ki, ri, vi, ko, ro, vo, n, shift, mask, hist, scan_tmp, s);
        cur ^= 1;
    }
    return cur;
}

// A mirror slab sorted by (column, row) in one or two passes (keys of at
// most 16 bits), the last pass putting rows and values into the full rows;
// the first pass reads its records straight from C_L, or, with extracted,
// from the record arrays key_a, row_a, val_a.  Returns the buffer with the
// sorted keys (for the column runs).
uint32_t* slab_sort_place(const SlabIo& io, int vbytes, int64_t nrec, int nbits, const int64_t* rec_rp, int64_t m,
                          bool extracted, uint32_t* key_a, uint32_t* key_b, uint32_t* row_a, uint32_t* row_b,
                          void* val_a, void* val_b, void* tmp, hipStream_t s) {
    if (nrec <= 0) return key_a;
    const int64_t ntiles = (nrec + kRTile - 1) / kRTile;
    uint32_t* hist = static_cast<uint32_t*>(tmp);
    const size_t hist_bytes = (size_t(ntiles) * kDigits * sizeof(uint32_t) + 255) & ~size_t(255);
    const size_t table_bytes = (size_t(ntiles + 1) * sizeof(int64_t) + 255) & ~size_t(255);
    int64_t* trow = reinterpret_cast<int64_t*>(static_cast<char*>(tmp) + hist_bytes);
    void* scan_tmp = static_cast<char*>(tmp) + hist_bytes + table_bytes;
    if (!extracted) tile_first_rows(rec_rp, m, kRTile, trow, s);
    int width[8];
    const int passes = digit_plan(nbits, width);
    const uint32_t m0 = (1u << width[0]) - 1u;
    uint32_t* out = key_b;
    auto go = [&](auto vb) {
        constexpr int VB = decltype(vb)::value;
        if (extracted) {
            if (passes == 1) {
                run_pass<VB, kSrcArrays, kOutPlace>(key_a, row_a, val_a, key_b, nullptr, nullptr, nrec, 0, m0, hist,
                                                    scan_tmp, s, nullptr, 0, nullptr, 0, 0, io);
            } else {
                run_pass<VB>(key_a, row_a, val_a, key_b, row_b, val_b, nrec, 0, m0, hist, scan_tmp, s);
                run_pass<VB, kSrcArrays, kOutPlace>(key_b, row_b, val_b, key_a, nullptr, nullptr, nrec, width[0],
                                                    (1u << width[1]) - 1u, hist, scan_tmp, s, nullptr, 0, nullptr, 0,
                                                    0, io);
                out = key_a;
            }
        } else if (passes == 1) {
            run_pass<VB, kSrcSlab, kOutPlace>(nullptr, nullptr, nullptr, key_b, nullptr, nullptr, nrec, 0, m0, hist,
                                              scan_tmp, s, rec_rp, m, trow, 0, 0, io);
        } else {
            run_pass<VB, kSrcSlab>(nullptr, nullptr, nullptr, key_a, row_a, val_a, nrec, 0, m0, hist, scan_tmp, s,
                                   rec_rp, m, trow, 0, 0, io);
            run_pass<VB, kSrcArrays, kOutPlace>(key_a, row_a, val_a, key_b, nullptr, nullptr, nrec, width[0],
                                                (1u << width[1]) - 1u, hist, scan_tmp, s, nullptr, 0, nullptr, 0, 0,
                                                io);
        }
    };
    if (vbytes == 8)
        go(std::integral_constant<int, 8>());
    else if (vbytes == 4)
        go(std::integral_constant<int, 4>());
    else
        go(std::integral_constant<int, 0>());
    return out;
}

}  // namespace spsyrk
