// Reference oracle for the local sparse SYRK: C_L = tril(A * A^T) in CSR.
//
// TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, single-threaded CPU
// statement of what the GPU library computes.  It shares no code, header,
// table or helper with the HIP library and must never be linked into it or
// called from its product path; only the tests, the smoke check and the
// benchmark's CPU-baseline leg load it.
//
// What it computes (paper Sec. II-A: C = A A^T for A in R^{m x n}; Sec. III-A:
// only the lower triangle of a diagonal block is formed; Sec. V-F, Eq. (spmv):
// the stored lower part includes the diagonal, C = C_L + C_L^T - D):
//
//   C_L(i, j) = sum_{k in S(i) and S(j)} A(i, k) * A(j, k),   0 <= j <= i < m,
//
// with S(r) the stored columns of row r.  An entry is stored iff S(i) and
// S(j) intersect (structure is the pattern product; computed zeros are kept).
// Rows keep A's order and columns ascend inside each row.
//
// The off-diagonal block (Sec. III-B, C_ij = sum_s A_is A_js^T) is the same
// formula over rows of A_i and rows of A_j with no triangle prune.
//
// A thin driver (syrk_sharded) runs the same per-row code on several threads,
// each taking blocks of consecutive rows, and joins the blocks in row order;
// it is there to time the oracle on all host cores and to check large
// results, and computes exactly what the single-threaded call does.
//
// Algorithm: Gustavson row by row.  A column-major copy of the right operand
// is built with a two-pass counting transpose (row ids come out ascending in
// each column), then for each output row a std::map keyed by output column
// accumulates the products in ascending k, and is emitted in key order.
//
// Semirings:
//   0  plus-times fp64  : accumulate in double.
//   1  plus-times fp32  : fp32 x fp32 products are exact in double; accumulate
//                         in double and round to float once at emit.  The sum
//                         of |products| is reported for the tolerance check.
//   2  count int32      : one per shared column (pattern only), uint32 wrap.
//   3  count -> Jaccard : c / (|a| + |b| - c) as one IEEE float division,
//                         |a|, |b| the stored lengths of the two rows.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <map>
#include <new>
#include <thread>
#include <vector>

namespace {

enum Semiring { F64 = 0, F32 = 1, COUNT = 2, JACCARD = 3 };

struct Acc {
    double sum = 0.0;
    double sum_abs = 0.0;
    uint32_t count = 0;
};

struct Result {
    int64_t nrows = 0;
    int64_t ncols = 0;
    std::vector<int64_t> row_ptr;
    std::vector<int32_t> col;
    std::vector<double> val;      // f64 value, or f32 value widened, or count / Jaccard
    std::vector<double> sum_abs;  // sum of |a*b| per entry
    std::vector<uint32_t> count;  // number of shared columns per entry
};

struct Csr {
    int64_t m, n;
    const int64_t* rp;
    const int32_t* ci;
    const void* v;
};

// 0 ok, 1 not canonical
int check_canonical(const Csr& A) {
    if (A.m < 0 || A.n < 0) return 1;
    if (A.rp[0] != 0) return 1;
    for (int64_t i = 0; i < A.m; ++i) {
        if (A.rp[i + 1] < A.rp[i]) return 1;
        for (int64_t e = A.rp[i]; e < A.rp[i + 1]; ++e) {
            if (A.ci[e] < 0 || A.ci[e] >= A.n) return 1;
            if (e > A.rp[i] && A.ci[e] <= A.ci[e - 1]) return 1;
        }
    }
    return 0;
}

double value_of(const Csr& A, int sr, int64_t e) {
    if (sr == F64) return static_cast<const double*>(A.v)[e];
    if (sr == F32) return static_cast<double>(static_cast<const float*>(A.v)[e]);
    return 1.0;
}

// Column-major copy of B (m_b x n): for column k, the rows holding k in
// ascending order, with their values.
struct Csc {
    std::vector<int64_t> ptr;
    std::vector<int32_t> row;
    std::vector<double> val;
};

Csc counting_transpose(const Csr& B, int sr) {
    Csc T;
    T.ptr.assign(static_cast<size_t>(B.n) + 1, 0);
    const int64_t nnz = B.rp[B.m];
    for (int64_t e = 0; e < nnz; ++e) T.ptr[B.ci[e] + 1]++;
    for (int64_t k = 0; k < B.n; ++k) T.ptr[k + 1] += T.ptr[k];
    T.row.resize(nnz);
    T.val.resize(nnz);
    std::vector<int64_t> next(T.ptr.begin(), T.ptr.end() - 1);
    for (int64_t r = 0; r < B.m; ++r) {
        for (int64_t e = B.rp[r]; e < B.rp[r + 1]; ++e) {
            const int64_t slot = next[B.ci[e]]++;
            T.row[slot] = static_cast<int32_t>(r);
            T.val[slot] = value_of(B, sr, e);
        }
    }
    return T;
}

void emit_row(Result& R, const std::map<int32_t, Acc>& acc, int sr, int64_t len_i, const Csr& B) {
    for (const auto& kv : acc) {
        const int32_t j = kv.first;
        const Acc& a = kv.second;
        R.col.push_back(j);
        R.sum_abs.push_back(a.sum_abs);
        R.count.push_back(a.count);
        if (sr == F64) {
            R.val.push_back(a.sum);
        } else if (sr == F32) {
            R.val.push_back(static_cast<double>(static_cast<float>(a.sum)));
        } else if (sr == COUNT) {
            R.val.push_back(static_cast<double>(static_cast<int32_t>(a.count)));
        } else {
            const int64_t len_j = B.rp[j + 1] - B.rp[j];
            const float c = static_cast<float>(a.count);
            const float d = static_cast<float>(len_i + len_j - static_cast<int64_t>(a.count));
            const float J = c / d;
            R.val.push_back(static_cast<double>(J));
        }
    }
}

// Output rows q in [q0, q1) of the product (row i = rows[q], or q), appended
// to R (R->row_ptr[q + 1] set relative to R's own entries).
// lower: right operand is A itself and only j <= i is kept.
void syrk_rows(bool lower, const Csr& A, const Csr& B, const Csc& T, int sr, const int64_t* rows, int64_t q0,
               int64_t q1, Result& R) {
    for (int64_t q = q0; q < q1; ++q) {
        const int64_t i = rows ? rows[q] : q;
        std::map<int32_t, Acc> acc;
        for (int64_t e = A.rp[i]; e < A.rp[i + 1]; ++e) {
            const int32_t k = A.ci[e];
            const double a = value_of(A, sr, e);
            for (int64_t p = T.ptr[k]; p < T.ptr[k + 1]; ++p) {
                const int32_t j = T.row[p];
                if (lower && j > i) break;  // column rows ascend: the rest is above the diagonal
                const double prod = a * T.val[p];
                Acc& s = acc[j];
                s.sum += prod;
                s.sum_abs += std::fabs(prod);
                s.count += 1u;
            }
        }
        emit_row(R, acc, sr, A.rp[i + 1] - A.rp[i], B);
        R.row_ptr[q - q0 + 1] = static_cast<int64_t>(R.col.size());
    }
}

// rows/nsel: optional subset of output rows (in the given order).
Result* syrk(bool lower, const Csr& A, const Csr& B, int sr, const int64_t* rows, int64_t nsel) {
    Result* R = new Result();
    const Csc T = counting_transpose(B, sr);
    const int64_t nout = rows ? nsel : A.m;
    R->nrows = nout;
    R->ncols = B.m;
    R->row_ptr.assign(static_cast<size_t>(nout) + 1, 0);
    syrk_rows(lower, A, B, T, sr, rows, 0, nout, *R);
    return R;
}

// The same rows computed by nthreads threads, each taking blocks of
// consecutive output rows from a shared counter; the blocks are joined in
// row order.  A driver for timing and for checking large results: every
// row goes through syrk_rows exactly as above.
Result* syrk_sharded(bool lower, const Csr& A, const Csr& B, int sr, const int64_t* rows, int64_t nsel,
                     int nthreads) {
    const Csc T = counting_transpose(B, sr);
    const int64_t nout = rows ? nsel : A.m;
    constexpr int64_t kBlockRows = 8192;
    const int64_t nblocks = (nout + kBlockRows - 1) / kBlockRows;
    std::vector<Result> part(static_cast<size_t>(nblocks));
    std::atomic<int64_t> next{0};
    std::atomic<bool> failed{false};
    auto work = [&]() {
        try {
            for (int64_t b = next++; b < nblocks && !failed; b = next++) {
                const int64_t q0 = b * kBlockRows, q1 = std::min(nout, q0 + kBlockRows);
                Result& P = part[static_cast<size_t>(b)];
                P.row_ptr.assign(static_cast<size_t>(q1 - q0) + 1, 0);
                syrk_rows(lower, A, B, T, sr, rows, q0, q1, P);
            }
        } catch (const std::bad_alloc&) {
            failed = true;
        }
    };
    std::vector<std::thread> pool;
    for (int t = 1; t < nthreads; ++t) pool.emplace_back(work);
    work();
    for (auto& th : pool) th.join();
    if (failed) throw std::bad_alloc();
    // join: block offsets, then every block copied into place (in parallel)
    Result* R = new Result();
    R->nrows = nout;
    R->ncols = B.m;
    R->row_ptr.assign(static_cast<size_t>(nout) + 1, 0);
    std::vector<size_t> base(static_cast<size_t>(nblocks) + 1, 0);
    for (int64_t b = 0; b < nblocks; ++b)
        base[static_cast<size_t>(b) + 1] = base[static_cast<size_t>(b)] + part[static_cast<size_t>(b)].col.size();
    const size_t total = base.back();
    R->col.resize(total);
    R->val.resize(total);
    R->sum_abs.resize(total);
    R->count.resize(total);
    next = 0;
    auto join = [&]() {
        for (int64_t b = next++; b < nblocks; b = next++) {
            Result& P = part[static_cast<size_t>(b)];
            const size_t o = base[static_cast<size_t>(b)];
            for (size_t r = 1; r < P.row_ptr.size(); ++r)
                R->row_ptr[static_cast<size_t>(b * kBlockRows) + r] = static_cast<int64_t>(o) + P.row_ptr[r];
            std::copy(P.col.begin(), P.col.end(), R->col.begin() + static_cast<std::ptrdiff_t>(o));
            std::copy(P.val.begin(), P.val.end(), R->val.begin() + static_cast<std::ptrdiff_t>(o));
            std::copy(P.sum_abs.begin(), P.sum_abs.end(), R->sum_abs.begin() + static_cast<std::ptrdiff_t>(o));
            std::copy(P.count.begin(), P.count.end(), R->count.begin() + static_cast<std::ptrdiff_t>(o));
            P = Result();  // release the block
        }
    };
    pool.clear();
    for (int t = 1; t < nthreads; ++t) pool.emplace_back(join);
    join();
    for (auto& th : pool) th.join();
    return R;
}

}  // namespace

extern "C" {

int oracle_check_canonical(int64_t m, int64_t n, const int64_t* rp, const int32_t* ci) {
    Csr A{m, n, rp, ci, nullptr};
    return check_canonical(A);
}

// mode 0: lower (B ignored), mode 1: offdiag A_i * A_j^T.  nthreads > 1
// computes the rows in blocks on that many threads (same rows, same values).
// Returns 0 on success, 1 not canonical, 2 shape mismatch, 3 out of memory.
int oracle_syrk_threads(int mode, int semiring,
                        int64_t m_a, int64_t n, const int64_t* rp_a, const int32_t* ci_a, const void* v_a,
                        int64_t m_b, int64_t n_b, const int64_t* rp_b, const int32_t* ci_b, const void* v_b,
                        const int64_t* rows, int64_t nsel, int nthreads, void** out) {
    *out = nullptr;
    Csr A{m_a, n, rp_a, ci_a, v_a};
    if (check_canonical(A)) return 1;
    Csr B = A;
    if (mode == 1) {
        B = Csr{m_b, n_b, rp_b, ci_b, v_b};
        if (n_b != n) return 2;
        if (check_canonical(B)) return 1;
    }
    if (rows) {
        for (int64_t q = 0; q < nsel; ++q)
            if (rows[q] < 0 || rows[q] >= m_a) return 2;
    }
    try {
        *out = nthreads > 1 ? syrk_sharded(mode == 0, A, B, semiring, rows, nsel, nthreads)
                            : syrk(mode == 0, A, B, semiring, rows, nsel);
    } catch (const std::bad_alloc&) {
        return 3;
    }
    return 0;
}

int oracle_syrk(int mode, int semiring,
                int64_t m_a, int64_t n, const int64_t* rp_a, const int32_t* ci_a, const void* v_a,
                int64_t m_b, int64_t n_b, const int64_t* rp_b, const int32_t* ci_b, const void* v_b,
                const int64_t* rows, int64_t nsel, void** out) {
    return oracle_syrk_threads(mode, semiring, m_a, n, rp_a, ci_a, v_a, m_b, n_b, rp_b, ci_b, v_b, rows, nsel, 1,
                               out);
}

// Full symmetric matrix from its stored lower part (Eq. (spmv): C = C_L + C_L^T - D):
// row i is the lower row i followed by the entries (r, i) of the strict lower
// part with r > i, in ascending r.  val_bytes is 4 or 8 (bits are copied).
// Returns 1 if an entry lies above the diagonal or the input is not canonical.
int oracle_mirror(int64_t m, const int64_t* rp, const int32_t* ci, const void* val, int val_bytes,
                  void** out) {
    *out = nullptr;
    Csr L{m, m, rp, ci, nullptr};
    if (check_canonical(L)) return 1;
    for (int64_t i = 0; i < m; ++i)
        for (int64_t e = rp[i]; e < rp[i + 1]; ++e)
            if (ci[e] > i) return 1;
    try {
        std::vector<std::vector<std::pair<int32_t, int64_t>>> full(static_cast<size_t>(m));
        for (int64_t i = 0; i < m; ++i)
            for (int64_t e = rp[i]; e < rp[i + 1]; ++e) full[i].push_back({ci[e], e});
        for (int64_t r = 0; r < m; ++r)
            for (int64_t e = rp[r]; e < rp[r + 1]; ++e)
                if (ci[e] < r) full[ci[e]].push_back({static_cast<int32_t>(r), e});
        Result* R = new Result();
        R->nrows = m;
        R->ncols = m;
        R->row_ptr.assign(static_cast<size_t>(m) + 1, 0);
        for (int64_t i = 0; i < m; ++i) {
            for (const auto& ce : full[i]) {
                R->col.push_back(ce.first);
                double bits = 0.0;  // raw bits carried through a double slot
                std::memcpy(&bits, static_cast<const char*>(val) + ce.second * val_bytes,
                            static_cast<size_t>(val_bytes));
                R->val.push_back(bits);
                R->sum_abs.push_back(0.0);
                R->count.push_back(0u);
            }
            R->row_ptr[i + 1] = static_cast<int64_t>(R->col.size());
        }
        *out = R;
    } catch (const std::bad_alloc&) {
        return 3;
    }
    return 0;
}

int64_t oracle_result_nrows(const void* h) { return static_cast<const Result*>(h)->nrows; }
int64_t oracle_result_nnz(const void* h) { return static_cast<int64_t>(static_cast<const Result*>(h)->col.size()); }

// Copy out.  val_kind: 0 -> double[], 1 -> float[], 2 -> int32[], 3 -> float[],
// 4 -> raw bytes (mirror; val_bytes given to oracle_mirror).  Any pointer may be null.
void oracle_result_copy(const void* h, int64_t* row_ptr, int32_t* col, void* val, int val_kind,
                        int val_bytes, double* sum_abs, uint32_t* count) {
    const Result* R = static_cast<const Result*>(h);
    const size_t nnz = R->col.size();
    if (row_ptr) std::memcpy(row_ptr, R->row_ptr.data(), R->row_ptr.size() * sizeof(int64_t));
    if (nnz == 0) return;  // an empty vector's data() may be null, and memcpy takes no null
    if (col) std::memcpy(col, R->col.data(), nnz * sizeof(int32_t));
    if (sum_abs) std::memcpy(sum_abs, R->sum_abs.data(), nnz * sizeof(double));
    if (count) std::memcpy(count, R->count.data(), nnz * sizeof(uint32_t));
    if (!val) return;
    for (size_t p = 0; p < nnz; ++p) {
        switch (val_kind) {
            case 0: static_cast<double*>(val)[p] = R->val[p]; break;
            case 1:
            case 3: static_cast<float*>(val)[p] = static_cast<float>(R->val[p]); break;
            case 2: static_cast<int32_t*>(val)[p] = static_cast<int32_t>(R->val[p]); break;
            default:
                std::memcpy(static_cast<char*>(val) + p * val_bytes, &R->val[p], static_cast<size_t>(val_bytes));
        }
    }
}

void oracle_result_free(void* h) { delete static_cast<Result*>(h); }

}  // extern "C"
