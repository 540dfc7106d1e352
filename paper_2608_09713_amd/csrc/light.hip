// Gustavson accumulation for rows with few products (row by row over A, the
// partners of each stored A(i,k) found in the column index of the right
// operand), batched: one workgroup takes 64 consecutive rows and handles them
// in sub-batches whose products fit in LDS.
//
// Accumulator: an ordered bucket sort in LDS.  Row r of a sub-batch owns
// nb_r = 2^ceil(log2(products_r)) buckets that split its column range
// [0, 2^bits) evenly, so bucket order is column order.  Products are counted
// per bucket, the counts scanned, the products scattered to their buckets,
// and inside each (small) bucket every product finds by comparison whether it
// is the first of its column (the leader), the leader's rank among the
// distinct columns of the bucket and, for values, the sum of its column's
// terms in product order.  A scan of the per-bucket distinct counts gives
// every leader its place in the output row, already in ascending column order.
//
// The symbolic pass writes the row lengths; the numeric pass repeats the same
// steps and writes columns and values at the scanned row offsets.  Rows whose
// products or entries exceed the LDS budget are handed to the dense-tile path.
#include "common.h"
#include "internal.h"
#include "lookup.h"

namespace spsyrk {
namespace {

constexpr int kRB = 64;        // rows per workgroup
constexpr int kECap = 512;     // entries per sub-batch
constexpr int kPCap = 1024;    // products per sub-batch (and the light-row limit)
constexpr int kBCap = 2 * kPCap + kRB;

template <int SR, bool NUM, bool LOWER>
__global__ __launch_bounds__(kBlock) void light_kernel(LightArgs a) {
    using Tr = SrTraits<SR>;
    using In = typename Tr::In;
    using Item = typename Tr::Item;
    constexpr bool kVal = (SR == kF64 || SR == kF32);
    constexpr bool kItem = Tr::kHasItem && NUM;

    __shared__ int64_t rp_s[kRB + 1];
    __shared__ uint32_t row_prod[kRB];
    __shared__ uint32_t row_nb[kRB];
    __shared__ uint32_t row_bb[kRB + 1];
    __shared__ uint8_t row_sh[kRB];
    __shared__ uint32_t ent_start[kECap];
    __shared__ uint32_t ent_len[kECap];
    __shared__ uint32_t ent_poff[kECap + 1];
    __shared__ uint8_t ent_row[kECap];
    __shared__ double ent_a[kVal && NUM ? kECap : 1];
    __shared__ uint32_t s_j[kPCap];
    __shared__ uint32_t s_rt[kPCap];
    __shared__ Item s_v[kItem ? kPCap : 1];
    __shared__ uint8_t s_lead[kPCap];
    __shared__ uint16_t s_rank[kPCap];
    __shared__ uint16_t s_cnt[(SR == kCount || SR == kJaccard) && NUM ? kPCap : 1];
    __shared__ uint32_t hist[kBCap + 1];
    __shared__ uint32_t ucnt[kBCap + 1];
    __shared__ uint32_t wt[kWavesPerBlock];
    __shared__ uint64_t wt64[kWavesPerBlock];
    __shared__ uint32_t nbuck_s;

    const int tid = threadIdx.x;
    const int64_t r0 = int64_t(blockIdx.x) * kRB;
    if (r0 >= a.m) return;
    const int nrows = int(min(int64_t(kRB), a.m - r0));
    for (int t = tid; t <= nrows; t += kBlock) rp_s[t] = a.rp[r0 + t];
    for (int t = tid; t < kRB; t += kBlock) row_prod[t] = 0;
    __syncthreads();

    const uint32_t* __restrict__ key = a.cx.key;
    const uint32_t rowmask = a.cx.rowbits >= 32 ? 0xffffffffu : ((1u << a.cx.rowbits) - 1u);
    const int jbits_right = bit_width_u64(a.m_right > 0 ? uint64_t(a.m_right - 1) : 0);
    uint64_t products_here = 0;

    int row = 0;
    while (row < nrows) {
        // entry window: rows [row, rend) holding at most kECap entries
        int rend = row;
        while (rend < nrows && rp_s[rend + 1] - rp_s[row] <= kECap) ++rend;
        if (rend == row) {
            if (!NUM && tid == 0) {
                const int h = atomicAdd(a.heavy_count, 1);
                a.heavy_rows[h] = int32_t(r0 + row);
            }
            ++row;
            continue;
        }
        const int64_t ebase = rp_s[row];
        const int ne = int(rp_s[rend] - ebase);
        for (int le = tid; le < ne; le += kBlock) {
            const int64_t e = ebase + le;
            // local row of e: last r in [row, rend) with rp_s[r] <= e
            int lo = row, hi = rend - 1;
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (rp_s[mid] <= e)
                    lo = mid;
                else
                    hi = mid - 1;
            }
            const uint32_t i = uint32_t(r0 + lo);
            uint32_t st, len;
            partner_run(key, a.cx.gptr, a.cx.gs, a.cx.rowbits, uint32_t(a.ci[e]), i, LOWER, st, len);
            ent_start[le] = st;
            ent_len[le] = len;
            ent_row[le] = uint8_t(lo);
            if constexpr (kVal && NUM) ent_a[le] = double(static_cast<const In*>(a.val)[e]);
            atomicAdd(&row_prod[lo], len);
        }
        __syncthreads();

        int ra = row;
        while (ra < rend) {
            if (row_prod[ra] > kPCap) {
                if (!NUM && tid == 0) {
                    const int h = atomicAdd(a.heavy_count, 1);
                    a.heavy_rows[h] = int32_t(r0 + ra);
                }
                ++ra;
                continue;
            }
            int rb = ra;
            uint32_t acc = 0;
            while (rb < rend && row_prod[rb] <= kPCap && acc + row_prod[rb] <= kPCap) {
                acc += row_prod[rb];
                ++rb;
            }
            const int nr = rb - ra;
            const int la = int(rp_s[ra] - ebase);
            const int lb = int(rp_s[rb] - ebase);
            const int nle = lb - la;

            // product offsets of the entries
            for (int x = tid; x < nle; x += kBlock) ent_poff[x] = ent_len[la + x];
            __syncthreads();
            const uint32_t P = block_exclusive_scan_array(ent_poff, nle, wt);
            if (tid == 0) ent_poff[nle] = P;
            // per-row buckets
            if (tid < kWave) {
                uint32_t nb = 0;
                if (tid < nr) {
                    const int r = ra + tid;
                    const uint32_t prod = row_prod[r];
                    int lognb = 0;
                    while ((1u << lognb) < prod) ++lognb;
                    nb = 1u << lognb;
                    const int64_t i = r0 + r;
                    const int jb = LOWER ? bit_width_u64(i > 0 ? uint64_t(i - 1) : 0) : jbits_right;
                    row_nb[tid] = nb;
                    row_sh[tid] = uint8_t(jb > lognb ? jb - lognb : 0);
                }
                const uint32_t inc = wave_inclusive_scan(nb);
                if (tid < nr) row_bb[tid] = inc - nb;
                if (tid == kWave - 1) nbuck_s = inc;
            }
            __syncthreads();
            const uint32_t B = nbuck_s;
            for (uint32_t b = tid; b <= B; b += kBlock) {
                hist[b] = 0;
                ucnt[b] = 0;
            }
            __syncthreads();

            // pass 1: bucket counts
            for (uint32_t t = tid; t < P; t += kBlock) {
                const int x = upper_bound_lds(ent_poff, 0, nle, t) - 1;
                const int le = la + x;
                const uint32_t pos = ent_start[le] + (t - ent_poff[x]);
                const uint32_t j = key[pos] & rowmask;
                const int rr = ent_row[le] - ra;
                atomicAdd(&hist[row_bb[rr] + (j >> row_sh[rr])], 1u);
            }
            __syncthreads();
            block_exclusive_scan_array(hist, int(B), wt);
            // pass 2: scatter into buckets
            for (uint32_t t = tid; t < P; t += kBlock) {
                const int x = upper_bound_lds(ent_poff, 0, nle, t) - 1;
                const int le = la + x;
                const uint32_t pos = ent_start[le] + (t - ent_poff[x]);
                const uint32_t j = key[pos] & rowmask;
                const int rr = ent_row[le] - ra;
                const uint32_t q = atomicAdd(&hist[row_bb[rr] + (j >> row_sh[rr])], 1u);
                s_j[q] = j;
                s_rt[q] = (uint32_t(rr) << 16) | t;
                if constexpr (kItem) {
                    if constexpr (SR == kJaccard)
                        s_v[q] = static_cast<const int32_t*>(a.cx.val)[pos];
                    else
                        s_v[q] = ent_a[le] * double(static_cast<const In*>(a.cx.val)[pos]);
                }
            }
            __syncthreads();
            // hist[b] is now the end of bucket b; its start is hist[b - 1]
            for (uint32_t q = tid; q < P; q += kBlock) {
                const uint32_t j = s_j[q];
                const uint32_t t = s_rt[q] & 0xffffu;
                const int rr = int(s_rt[q] >> 16);
                const uint32_t b = row_bb[rr] + (j >> row_sh[rr]);
                const uint32_t lo = b ? hist[b - 1] : 0u, hi = hist[b];
                uint8_t lead = 1;
                for (uint32_t u = lo; u < hi; ++u)
                    if (s_j[u] == j && (s_rt[u] & 0xffffu) < t) lead = 0;
                s_lead[q] = lead;
            }
            __syncthreads();
            for (uint32_t q = tid; q < P; q += kBlock) {
                if (!s_lead[q]) continue;
                const uint32_t j = s_j[q];
                const uint32_t t = s_rt[q] & 0xffffu;
                const int rr = int(s_rt[q] >> 16);
                const uint32_t b = row_bb[rr] + (j >> row_sh[rr]);
                const uint32_t lo = b ? hist[b - 1] : 0u, hi = hist[b];
                uint32_t rank = 0, cnt = 0;
                for (uint32_t u = lo; u < hi; ++u) {
                    const uint32_t ju = s_j[u];
                    rank += (s_lead[u] && ju < j) ? 1u : 0u;
                    cnt += ju == j ? 1u : 0u;
                }
                s_rank[q] = uint16_t(rank);
                atomicAdd(&ucnt[b], 1u);
                if constexpr (NUM) {
                    if constexpr (kVal) {
                        // terms of column j in product order (the order of k along row i)
                        double sum = s_v[q];
                        uint32_t last = t;
                        for (uint32_t c = 1; c < cnt; ++c) {
                            uint32_t best = 0xffffffffu, bu = lo;
                            for (uint32_t u = lo; u < hi; ++u) {
                                const uint32_t tu = s_rt[u] & 0xffffu;
                                if (s_j[u] == j && tu > last && tu < best) {
                                    best = tu;
                                    bu = u;
                                }
                            }
                            sum += s_v[bu];
                            last = best;
                        }
                        s_v[q] = sum;
                    } else {
                        s_cnt[q] = uint16_t(cnt);
                    }
                }
            }
            __syncthreads();
            const uint32_t U = block_exclusive_scan_array(ucnt, int(B), wt);
            if (tid == 0) ucnt[B] = U;
            __syncthreads();
            // row lengths, diagonal
            if (tid < nr) {
                const int r = ra + tid;
                const int64_t i = r0 + r;
                const int64_t rowlen = rp_s[r + 1] - rp_s[r];
                const uint32_t offn = ucnt[row_bb[tid] + row_nb[tid]] - ucnt[row_bb[tid]];
                const bool diag = LOWER && rowlen > 0;
                if constexpr (!NUM) {
                    a.row_nnz[i] = int64_t(offn) + (diag ? 1 : 0);
                } else if (diag) {
                    const int64_t p = a.c_rp[i] + offn;
                    a.c_ci[p] = int32_t(i);
                    using Out = typename Tr::Out;
                    Out dv;
                    if constexpr (kVal) {
                        double s = 0.0;
                        const int ea = int(rp_s[r] - ebase), eb = int(rp_s[r + 1] - ebase);
                        for (int le = ea; le < eb; ++le) s += ent_a[le] * ent_a[le];
                        dv = Out(s);
                    } else if constexpr (SR == kCount) {
                        dv = int32_t(rowlen);
                    } else {
                        dv = jaccard(int32_t(rowlen), rowlen, rowlen);
                    }
                    static_cast<Out*>(a.c_val)[p] = dv;
                }
            }
            if constexpr (NUM) {
                using Out = typename Tr::Out;
                for (uint32_t q = tid; q < P; q += kBlock) {
                    if (!s_lead[q]) continue;
                    const uint32_t j = s_j[q];
                    const int rr = int(s_rt[q] >> 16);
                    const uint32_t b = row_bb[rr] + (j >> row_sh[rr]);
                    const int64_t i = r0 + ra + rr;
                    const int64_t p = a.c_rp[i] + (ucnt[b] - ucnt[row_bb[rr]]) + s_rank[q];
                    a.c_ci[p] = int32_t(j);
                    Out ov;
                    if constexpr (kVal) {
                        ov = Out(s_v[q]);
                    } else if constexpr (SR == kCount) {
                        ov = int32_t(s_cnt[q]);
                    } else {
                        ov = jaccard(int32_t(s_cnt[q]), rp_s[ra + rr + 1] - rp_s[ra + rr], s_v[q]);
                    }
                    static_cast<Out*>(a.c_val)[p] = ov;
                }
            }
            products_here += P;
            __syncthreads();
            ra = rb;
        }
        __syncthreads();
        row = rend;
    }
    if (!NUM && tid == 0 && products_here) atomicAdd(a.products, (unsigned long long)products_here);
    (void)wt64;
}

template <int SR, bool NUM>
void launch(const LightArgs& a, hipStream_t s) {
    const unsigned nb = unsigned((a.m + kRB - 1) / kRB);
    if (nb == 0) return;
    if (a.lower)
        light_kernel<SR, NUM, true><<<nb, kBlock, 0, s>>>(a);
    else
        light_kernel<SR, NUM, false><<<nb, kBlock, 0, s>>>(a);
}

template <bool NUM>
void dispatch(const LightArgs& a, hipStream_t s) {
    switch (a.sr) {
        case kF64: launch<kF64, NUM>(a, s); break;
        case kF32: launch<kF32, NUM>(a, s); break;
        case kCount: launch<kCount, NUM>(a, s); break;
        default: launch<kJaccard, NUM>(a, s); break;
    }
}

}  // namespace

void light_symbolic(const LightArgs& a, hipStream_t s) { dispatch<false>(a, s); }
void light_numeric(const LightArgs& a, hipStream_t s) { dispatch<true>(a, s); }

}  // namespace spsyrk
