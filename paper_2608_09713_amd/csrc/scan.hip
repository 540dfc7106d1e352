// Device-wide exclusive prefix sums (three launches: tile reduce, scan of
// tile sums in one workgroup, tile scan with carry-in; one launch for arrays
// of at most four tiles).
#include "common.h"
#include "internal.h"

namespace spsyrk {
namespace {

constexpr int kItems = 16;
constexpr int kTile = kBlock * kItems;

template <typename T>
__global__ __launch_bounds__(kBlock) void tile_reduce(const T* __restrict__ in, int64_t n, T* __restrict__ sums) {
    __shared__ T wt[kWavesPerBlock];
    const int64_t base = int64_t(blockIdx.x) * kTile;
    T s = 0;
#pragma unroll
    for (int k = 0; k < kItems; ++k) {
        int64_t i = base + int64_t(k) * kBlock + threadIdx.x;
        if (i < n) s += in[i];
    }
    s = wave_reduce_sum(s);
    if (lane_id() == 0) wt[threadIdx.x / kWave] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        T t = 0;
        for (int w = 0; w < kWavesPerBlock; ++w) t += wt[w];
        sums[blockIdx.x] = t;
    }
}

// exclusive scan of nb tile sums in place by one workgroup; total -> *total
template <typename T>
__global__ __launch_bounds__(kBlock) void scan_sums(T* __restrict__ sums, int64_t nb, T* __restrict__ total) {
    __shared__ T wt[kWavesPerBlock];
    T carry = 0;
    for (int64_t base = 0; base < nb; base += kTile) {
        // each thread takes kItems consecutive sums
        T v[kItems];
        T s = 0;
#pragma unroll
        for (int k = 0; k < kItems; ++k) {
            int64_t i = base + int64_t(threadIdx.x) * kItems + k;
            v[k] = i < nb ? sums[i] : T(0);
            s += v[k];
        }
        T tot;
        T off = block_exclusive_scan(s, wt, &tot);
        off += carry;
#pragma unroll
        for (int k = 0; k < kItems; ++k) {
            int64_t i = base + int64_t(threadIdx.x) * kItems + k;
            if (i < nb) sums[i] = off;
            off += v[k];
        }
        carry += tot;
        __syncthreads();
    }
    if (threadIdx.x == 0 && total) *total = carry;
}

// Exclusive scan of the tile at base (kTile values of in, zero past n) into
// out, starting from carry; returns the tile's sum.  The tile is read whole
// into LDS before any of it is written, so in may equal out.
template <typename T>
__device__ inline T scan_tile(const T* __restrict__ in, T* __restrict__ out, int64_t n, int64_t base, T carry,
                              T* buf, T* wt) {
    // coalesced loads into LDS, then a blocked arrangement: thread t holds
    // kItems consecutive elements
#pragma unroll
    for (int k = 0; k < kItems; ++k) {
        const int64_t i = base + int64_t(k) * kBlock + threadIdx.x;
        buf[k * kBlock + threadIdx.x] = i < n ? in[i] : T(0);
    }
    __syncthreads();
    T v[kItems];
    T s = 0;
#pragma unroll
    for (int k = 0; k < kItems; ++k) {
        v[k] = buf[threadIdx.x * kItems + k];
        s += v[k];
    }
    T tot;
    T off = block_exclusive_scan(s, wt, &tot) + carry;
#pragma unroll
    for (int k = 0; k < kItems; ++k) {
        buf[threadIdx.x * kItems + k] = off;
        off += v[k];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kItems; ++k) {
        const int64_t i = base + int64_t(k) * kBlock + threadIdx.x;
        if (i < n) out[i] = buf[k * kBlock + threadIdx.x];
    }
    __syncthreads();  // (buf is reused by the next tile)
    return tot;
}

template <typename T>
__global__ __launch_bounds__(kBlock) void tile_scan(const T* __restrict__ in, T* __restrict__ out, int64_t n,
                                                    const T* __restrict__ sums) {
    __shared__ T wt[kWavesPerBlock];
    __shared__ T buf[kTile];
    (void)scan_tile(in, out, n, int64_t(blockIdx.x) * kTile, sums[blockIdx.x], buf, wt);
}

// up to kOneBlockTiles tiles scanned by one workgroup, tile after tile with
// the carry (one launch instead of three for short arrays); total -> *total
constexpr int64_t kOneBlockTiles = 4;
template <typename T>
__global__ __launch_bounds__(kBlock) void scan_one_block(const T* __restrict__ in, T* __restrict__ out, int64_t n,
                                                         T* __restrict__ total) {
    __shared__ T wt[kWavesPerBlock];
    __shared__ T buf[kTile];
    T carry = 0;
    for (int64_t base = 0; base < n; base += kTile) carry += scan_tile(in, out, n, base, carry, buf, wt);
    if (total && threadIdx.x == 0) *total = carry;
}

template <typename T>
void scan_impl(const T* in, T* out, int64_t n, T* total, void* tmp, hipStream_t s) {
    const int64_t nb = (n + kTile - 1) / kTile;
    T* sums = static_cast<T*>(tmp);
    if (nb == 0) {
        if (total) (void)hipMemsetAsync(total, 0, sizeof(T), s);
        return;
    }
    if (nb <= kOneBlockTiles) {
        scan_one_block<T><<<1, kBlock, 0, s>>>(in, out, n, total);
        return;
    }
    tile_reduce<T><<<dim3(unsigned(nb)), dim3(kBlock), 0, s>>>(in, n, sums);
    scan_sums<T><<<1, kBlock, 0, s>>>(sums, nb, total);
    tile_scan<T><<<dim3(unsigned(nb)), dim3(kBlock), 0, s>>>(in, out, n, sums);
}

}  // namespace

size_t scan_tmp_bytes(int64_t n) { return size_t((n + kTile - 1) / kTile + 1) * sizeof(int64_t); }

void scan_u32(const uint32_t* in, uint32_t* out, int64_t n, uint32_t* total, void* tmp, hipStream_t s) {
    scan_impl<uint32_t>(in, out, n, total, tmp, s);
}

void scan_i64(const int64_t* in, int64_t* out, int64_t n, int64_t* total, void* tmp, hipStream_t s) {
    scan_impl<int64_t>(in, out, n, total, tmp, s);
}

}  // namespace spsyrk
