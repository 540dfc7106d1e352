// Device and host helpers shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace spsyrk {

constexpr int kWave = 64;        // gfx950 wavefront width
constexpr int kBlock = 256;      // threads per workgroup used by most kernels
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kXcds = 8;         // XCDs of the chip; workgroups are dealt to them round-robin

// error bits raised by validation kernels (OR-ed into one device word)
enum ErrBits : uint32_t {
    kErrRowPtr = 1u,        // row_ptr not monotone / wrong ends
    kErrColRange = 2u,      // column id outside [0, ncols)
    kErrColOrder = 4u,      // column ids not strictly increasing within a row
    kErrUpper = 8u,         // entry above the diagonal (mirror input)
};

// Debug checks, compiled only with -DSPSYRK_DEBUG=1.  A kernel that finds one
// of its invariants broken ORs the check's bit into a device word of its
// translation unit and goes on (no trap, so a broken check cannot take the
// device down); spsyrk_debug_flags() collects and clears every unit's word.
enum DbgBits : uint32_t {
    kDbgCompactOut = 1u,     // compaction: destination outside [0, nnz(C))
    kDbgHeavyOut = 2u,       // heavy rows: an output slot outside the row's range of C
    kDbgHeavyCount = 4u,     // heavy rows: the numeric pass found more columns than the symbolic pass
    kDbgReadFailed = 1u << 31,  // the host could not read a unit's word
};
namespace dbg {
using Reader = uint32_t (*)();
void add_reader(Reader r);  // registers a unit's reader (api.hip)
#if defined(SPSYRK_DEBUG) && SPSYRK_DEBUG
static __device__ unsigned word;
static uint32_t read_and_clear() {
    void* p = nullptr;
    uint32_t v = 0, z = 0;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(word)) != hipSuccess) return kDbgReadFailed;
    if (hipMemcpy(&v, p, sizeof v, hipMemcpyDeviceToHost) != hipSuccess) return kDbgReadFailed;
    if (hipMemcpy(p, &z, sizeof z, hipMemcpyHostToDevice) != hipSuccess) return kDbgReadFailed;
    return v;
}
[[maybe_unused]] static const bool registered = (add_reader(&read_and_clear), true);
#endif
}  // namespace dbg
#if defined(SPSYRK_DEBUG) && SPSYRK_DEBUG
#define SPSYRK_CHECK(cond, bit) \
    do {                        \
        if (!(cond)) atomicOr(&::spsyrk::dbg::word, uint32_t(bit)); \
    } while (0)
#else
#define SPSYRK_CHECK(cond, bit) \
    do {                        \
    } while (0)
#endif

// number of bits needed to write x (0 -> 0)
__host__ __device__ inline int bit_width_u64(uint64_t x) { return x ? 64 - __builtin_clzll(x) : 0; }

__device__ inline int lane_id() { return __lane_id(); }

// 16 bytes read once: a streamed load that does not displace cached lines
__device__ inline uint4 nt_load4(const void* p) {
    typedef unsigned int v4 __attribute__((ext_vector_type(4)));
    const v4 v = __builtin_nontemporal_load(reinterpret_cast<const v4*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

// a write not read again by this kernel: a streamed store, which leaves the
// caches to the kernel's scattered writes (those merge there into fuller lines)
template <typename T>
__device__ inline void nt_store(T v, T* p) {
    __builtin_nontemporal_store(v, p);
}

__device__ inline uint64_t lanemask_lt() { return (uint64_t(1) << lane_id()) - 1; }

// inclusive scan across a wavefront (64 lanes)
template <typename T>
__device__ inline T wave_inclusive_scan(T v) {
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        T u = __shfl_up(v, d, kWave);
        if (lane_id() >= d) v += u;
    }
    return v;
}

template <typename T>
__device__ inline T wave_reduce_sum(T v) {
#pragma unroll
    for (int d = kWave / 2; d > 0; d >>= 1) v += __shfl_xor(v, d, kWave);
    return v;
}

template <typename T>
__device__ inline T wave_reduce_max(T v) {
#pragma unroll
    for (int d = kWave / 2; d > 0; d >>= 1) {
        T u = __shfl_xor(v, d, kWave);
        v = u > v ? u : v;
    }
    return v;
}

// Exclusive scan of a block of NT values, one per thread.  `warp_tot` is LDS
// scratch of NT / kWave entries.  Returns the exclusive prefix of this thread
// and writes the block total to *total (all threads).
template <typename T, int NT = kBlock>
__device__ inline T block_exclusive_scan(T v, T* warp_tot, T* total) {
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    T inc = wave_inclusive_scan(v);
    if (lane == kWave - 1) warp_tot[w] = inc;
    __syncthreads();
    T off = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < NT / kWave; ++i) {
        T t = warp_tot[i];
        if (i < w) off += t;
        tot += t;
    }
    __syncthreads();
    *total = tot;
    return off + inc - v;
}

// maximum of v over the threads before this one in the workgroup (0 for the
// first thread); *all gets the maximum over every thread
__device__ inline uint32_t block_exclusive_max(uint32_t v, uint32_t* wt, uint32_t* all) {
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    uint32_t inc = v;
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const uint32_t u = __shfl_up(inc, d, kWave);
        if (lane >= d) inc = max(inc, u);
    }
    if (lane == kWave - 1) wt[w] = inc;
    __syncthreads();
    uint32_t before = 0, mx = 0;
#pragma unroll
    for (int q = 0; q < kWavesPerBlock; ++q) {
        const uint32_t t = wt[q];
        if (q < w) before = max(before, t);
        mx = max(mx, t);
    }
    __syncthreads();
    const uint32_t prev = __shfl_up(inc, 1, kWave);
    if (lane > 0) before = max(before, prev);
    *all = mx;
    return before;
}

// Exclusive scan in place of an LDS array of length n (any n) by the whole
// block of NT threads; returns the total.  `warp_tot` is LDS scratch of
// NT / kWave entries.
template <typename T, int NT = kBlock>
__device__ inline T block_exclusive_scan_array(T* a, int n, T* warp_tot) {
    const int per = (n + NT - 1) / NT;
    const int lo = min(n, int(threadIdx.x) * per);
    const int hi = min(n, lo + per);
    T s = 0;
    for (int i = lo; i < hi; ++i) s += a[i];
    T tot;
    T off = block_exclusive_scan<T, NT>(s, warp_tot, &tot);
    for (int i = lo; i < hi; ++i) {
        T x = a[i];
        a[i] = off;
        off += x;
    }
    __syncthreads();
    return tot;
}

// first index in [lo, hi) with a[idx] > x (a non-decreasing), else hi
template <typename T>
__device__ inline int upper_bound_lds(const T* a, int lo, int hi, T x) {
    while (lo < hi) {
        int mid = (lo + hi) >> 1;
        if (a[mid] <= x)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

// first index in [lo, hi) with key[idx] >= x, for non-decreasing uint32 keys in global memory
__device__ inline int64_t lower_bound_u32(const uint32_t* key, int64_t lo, int64_t hi, uint64_t x) {
    while (lo < hi) {
        int64_t mid = (lo + hi) >> 1;
        if (uint64_t(key[mid]) < x)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

}  // namespace spsyrk
