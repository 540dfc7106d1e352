// C-ABI entry points: argument checks, device-side validation, workspace and
// output allocation through the caller's allocator, and the kernel sequence.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"
#include "internal.h"
#include "spsyrk.h"

using namespace spsyrk;

uint32_t spsyrk::run_radix(int64_t positions) {
    const uint64_t p1 = uint64_t(positions > 0 ? positions : 0) + 1;
    uint64_t r = (uint64_t(1) << 32) / p1;
    if (r > (uint64_t(1) << 16)) r = uint64_t(1) << 16;
    if (r < 8) r = 1;
    if (const char* e = std::getenv("SPSYRK_RUN_RADIX")) {
        const long long want = std::atoll(e);
        r = want <= 1 ? 1 : (uint64_t(want) < r ? uint64_t(want) : r);
    }
    return uint32_t(r);
}

namespace {

thread_local std::string g_detail;
thread_local spsyrk_stats g_stats;
thread_local bool g_stats_valid = false;
// the two-pass kernels (symbolic, then numeric, partner runs looked up in a
// directory) instead of the single pass, for both calls (SPSYRK_TWO_PASS=1,
// read at every call; used to cross-check the two implementations)
bool two_pass() {
    const char* e = std::getenv("SPSYRK_TWO_PASS");
    return e && e[0] == '1';
}

// packed staging of count and Jaccard outputs where it fits (SPSYRK_PACK_STAGING=0
// turns it off; read at every call)
bool pack_staging() {
    const char* e = std::getenv("SPSYRK_PACK_STAGING");
    return !(e && e[0] == '0');
}

constexpr int64_t kLimit = int64_t(1) << 31;

void set_detail(const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_detail = buf;
}

struct Fail {
    spsyrk_status st;
};

#define HIPCHK(call)                                                                          \
    do {                                                                                      \
        hipError_t e_ = (call);                                                               \
        if (e_ != hipSuccess) {                                                               \
            set_detail("%s failed: %s (%s:%d)", #call, hipGetErrorString(e_), __FILE__, __LINE__); \
            throw Fail{SPSYRK_ERR_HIP};                                                       \
        }                                                                                     \
    } while (0)

// Allocations of one call.  Workspace is released at the end of the call
// (stream-ordered); outputs are released only if the call fails.
class Arena {
   public:
    Arena(const spsyrk_allocator* al, hipStream_t s) : al_(al), s_(s) {}
    bool touched() const { return touched_; }
    ~Arena() { release_all(); }

    // Allocate count blocks of the given size ahead of the gets that will
    // take them (any later get of that size takes one), so that those gets
    // cost the host nothing at a point where the device waits on it.
    void reserve(size_t bytes, int count = 1) {
        bytes = round(bytes);
        for (int i = 0; i < count; ++i) reserved_.push_back({raw(bytes), bytes});
    }

    void* get(size_t bytes, bool output = false) {
        touched_ = true;
        bytes = round(bytes);
        for (auto& r : reserved_)
            if (r.p && r.bytes == bytes) {
                void* p = r.p;
                r.p = nullptr;
                (output ? outputs_ : work_).push_back(p);
                return p;
            }
        void* p = raw(bytes);
        (output ? outputs_ : work_).push_back(p);
        return p;
    }
    template <typename T>
    T* get_t(int64_t count, bool output = false) {
        return static_cast<T*>(get(size_t(count) * sizeof(T), output));
    }
    void release(void* p) {
        for (auto& q : work_)
            if (q == p) {
                free_one(q);
                q = nullptr;
            }
    }
    // keep a work allocation past the call (it becomes the caller's, like an output)
    void* keep(void* p) {
        for (auto& q : work_)
            if (q == p) {
                q = nullptr;
                outputs_.push_back(p);
            }
        return p;
    }
    // release an allocation made as an output (an intermediate result)
    void release_output(void* p) {
        for (auto& q : outputs_)
            if (q == p) {
                free_one(q);
                q = nullptr;
            }
    }
    void keep_outputs() { outputs_.clear(); }
    void release_all() {
        for (void* p : work_)
            if (p) free_one(p);
        for (void* p : outputs_)
            if (p) free_one(p);
        for (auto& r : reserved_)
            if (r.p) free_one(r.p);
        work_.clear();
        outputs_.clear();
        reserved_.clear();
    }

   private:
    struct Reserved {
        void* p;
        size_t bytes;
    };
    static size_t round(size_t bytes) { return bytes == 0 ? 256 : (bytes + 255) & ~size_t(255); }
    void* raw(size_t bytes) {
        void* p = nullptr;
        if (al_ && al_->alloc) {
            p = al_->alloc(al_->ctx, bytes);
        } else {
            hipError_t e = hipMallocAsync(&p, bytes, s_);
            if (e != hipSuccess) p = nullptr;
        }
        if (!p) {
            set_detail("allocation of %zu bytes failed", bytes);
            throw Fail{SPSYRK_ERR_OOM};
        }
        return p;
    }
    void free_one(void* p) {
        if (al_ && al_->free)
            al_->free(al_->ctx, p);
        else if (!al_)
            (void)hipFreeAsync(p, s_);
    }
    const spsyrk_allocator* al_;
    hipStream_t s_;
    std::vector<void*> work_, outputs_;
    std::vector<Reserved> reserved_;
    bool touched_ = false;
};

// ---- phase timing: event pairs recorded on the call's stream
struct PhaseMark {
    int phase;
    hipEvent_t a, b;
};
thread_local bool g_timing = false;
thread_local uint32_t g_phase_mask = 0;  // bit p: phase p is timed
thread_local std::vector<PhaseMark> g_marks;
// events of finished marks, reused so that a timed call creates none
thread_local std::vector<hipEvent_t> g_event_pool;

hipEvent_t pooled_event() {
    if (!g_event_pool.empty()) {
        hipEvent_t e = g_event_pool.back();
        g_event_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    return hipEventCreate(&e) == hipSuccess ? e : nullptr;
}

void pool_event(hipEvent_t e) {
    if (e) g_event_pool.push_back(e);
}

using Phase = PhaseTimer;

// small block of device scalars read back at the synchronisation points
struct Ctl {
    uint32_t err;
    int32_t heavy_count;
    unsigned long long products;
    int64_t total;
    int64_t nkept;
    int64_t total2;
    int32_t queue;
    uint32_t err2;  // validation flags of the second operand (off the diagonal)
    unsigned long long light_cap;
    unsigned long long heavy_sums[2];  // entries of A and output entries of the heavy rows
    unsigned long long chunk_counter;
    unsigned long long maxlen;  // largest row length of the left operand
    int64_t pad[1];
};

struct HostCtl {
    Ctl* h = nullptr;
    hipEvent_t ev = nullptr;  // recorded after the copy into h
    HostCtl() {
        if (hipHostMalloc(reinterpret_cast<void**>(&h), sizeof(Ctl), hipHostMallocDefault) != hipSuccess) h = nullptr;
        if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess) ev = nullptr;
    }
    ~HostCtl() {
        if (h) (void)hipHostFree(h);
        if (ev) (void)hipEventDestroy(ev);
    }
};

HostCtl& host_ctl() {
    thread_local HostCtl pin;
    if (!pin.h || !pin.ev) {
        set_detail("pinned host buffer unavailable");
        throw Fail{SPSYRK_ERR_HIP};
    }
    return pin;
}

// Enqueue the copy of the control block to the host; ctl_wait returns it
// once the copy is done, while the work enqueued after the copy may still
// run.  (One copy in flight per thread: every ctl_fetch is followed by its
// ctl_wait before the next.)
void ctl_fetch(const Ctl* d, hipStream_t s) {
    HostCtl& pin = host_ctl();
    HIPCHK(hipMemcpyAsync(pin.h, d, sizeof(Ctl), hipMemcpyDeviceToHost, s));
    HIPCHK(hipEventRecord(pin.ev, s));
}

Ctl ctl_wait() {
    HostCtl& pin = host_ctl();
    // polled rather than blocked on: the waits are short, and a blocked
    // thread resumes some microseconds after the event, with the device idle
    hipError_t e;
    while ((e = hipEventQuery(pin.ev)) == hipErrorNotReady) {
    }
    HIPCHK(e);
    return *pin.h;
}

Ctl read_ctl(const Ctl* d, hipStream_t s) {
    ctl_fetch(d, s);
    return ctl_wait();
}

void check_launch() {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) {
        set_detail("kernel launch failed: %s", hipGetErrorString(e));
        throw Fail{SPSYRK_ERR_HIP};
    }
}

void check_input(const spsyrk_csr* A, int sr, bool need_values, const char* name, int64_t nnz_limit = kLimit) {
    if (!A) {
        set_detail("%s is null", name);
        throw Fail{SPSYRK_ERR_INVALID_ARG};
    }
    if (A->nrows < 0 || A->ncols < 0 || A->nnz < 0) {
        set_detail("%s has a negative size", name);
        throw Fail{SPSYRK_ERR_INVALID_ARG};
    }
    if (A->nrows >= kLimit || A->ncols >= kLimit || A->nnz >= nnz_limit) {
        set_detail("%s: nrows and ncols must be below 2^31 and nnz below %lld", name, (long long)nnz_limit);
        throw Fail{SPSYRK_ERR_SHAPE};
    }
    if (!A->row_ptr || (A->nnz > 0 && !A->col_idx)) {
        set_detail("%s: null row_ptr or col_idx", name);
        throw Fail{SPSYRK_ERR_INVALID_ARG};
    }
    if (need_values && A->nnz > 0 && !A->values && (sr == kF64 || sr == kF32)) {
        set_detail("%s: values are required for plus-times semirings", name);
        throw Fail{SPSYRK_ERR_INVALID_ARG};
    }
}

void check_semiring(int sr) {
    if (sr < 0 || sr > 3) {
        set_detail("unknown semiring %d", sr);
        throw Fail{SPSYRK_ERR_INVALID_ARG};
    }
}

DevCsr dev(const spsyrk_csr* A) {
    DevCsr d;
    d.m = A->nrows;
    d.n = A->ncols;
    d.nnz = A->nnz;
    d.rp = A->row_ptr;
    d.ci = A->col_idx;
    d.v = A->values;
    return d;
}

// Enqueue the validation of A, its flags into *err (zeroed beforehand);
// check_valid takes them from a later read of the control block.
// keep_rows (optional, validate_tmp_bytes(nnz)): the validation's table of
// tile rows is left there for later kernels (tiles of kRadixTile entries)
void validate_enqueue(const DevCsr& A, bool upper_forbidden, Arena& ar, uint32_t* err, hipStream_t s,
                      const FirstHist* fh = nullptr, void* keep_rows = nullptr) {
    void* vtmp = keep_rows ? keep_rows : ar.get(validate_tmp_bytes(A.nnz));
    validate_csr(A, upper_forbidden, err, vtmp, s, fh);
    check_launch();
    if (!keep_rows) ar.release(vtmp);  // (stream-ordered: later work may reuse it)
}

void check_valid(uint32_t err, const char* name) {
    if (err) {
        set_detail("%s is not canonical CSR (flags 0x%x:%s%s%s%s)", name, err, (err & kErrRowPtr) ? " row_ptr" : "",
                   (err & kErrColRange) ? " column-range" : "", (err & kErrColOrder) ? " column-order" : "",
                   (err & kErrUpper) ? " above-diagonal" : "");
        throw Fail{SPSYRK_ERR_NOT_CANONICAL};
    }
}

void validate(const DevCsr& A, bool upper_forbidden, Arena& ar, Ctl* ctl, hipStream_t s, const char* name,
              const FirstHist* fh = nullptr, void* keep_rows = nullptr) {
    validate_enqueue(A, upper_forbidden, ar, &ctl->err, s, fh, keep_rows);
    check_valid(read_ctl(ctl, s).err, name);
}

// Build the column index of B (sorted by column, packed keys, directory).
// With run (zeroed beforehand; lower mode) every entry's partner run is written.
// need_dir: build the group directory for partner-run lookups.
// ccount (zeroed, B.n entries, with no directory only): the entries of every
// column, written when the local sort builds the index (*counted is then set).
// vsrc (N entries): the entry of B behind every position of the index.
ColIndex build_index(const DevCsr& B, bool drop_last, int sr, Arena& ar, Ctl* ctl, hipStream_t s,
                     const RunTab* run = nullptr, bool need_dir = true, uint32_t* ccount = nullptr, bool* counted = nullptr,
                     uint32_t* vsrc = nullptr, uint32_t* hist1 = nullptr, const int64_t* trow1 = nullptr) {
    ColIndex cx;
    cx.n = B.n;
    cx.m = B.m;
    cx.rowbits = bit_width_u64(B.m > 1 ? uint64_t(B.m - 1) : 1);
    const int64_t N = B.nnz;
    // about 16 entries per directory group, limited by the key width
    int gs = 0;
    if (B.n > 0) {
        const double target = 16.0 * double(B.n) / double(N > 0 ? N : 1);
        while (gs < 31 && double(int64_t(1) << (gs + 1)) <= target) ++gs;
    }
    const int maxgs = 32 - cx.rowbits;
    if (gs > maxgs) gs = maxgs;
    const int nbits_n = bit_width_u64(B.n > 1 ? uint64_t(B.n - 1) : 0);
    if (gs > nbits_n) gs = nbits_n;
    // with every partner run given nothing is ever looked up: no directory,
    // and the keys hold the row only
    const bool runs_given = run != nullptr || !need_dir;
    if (runs_given) gs = 0;
    cx.gs = gs;
    cx.ngroups = B.n > 0 ? ((B.n + (int64_t(1) << gs) - 1) >> gs) : 0;
    const int vb = (sr == kF64) ? 8 : (sr == kF32 ? 4 : 0);
    const int vb_out = csc_value_bytes(sr);

    cx.gptr = runs_given ? nullptr : ar.get_t<uint32_t>(cx.ngroups + 1);
    cx.key = ar.get_t<uint32_t>(N > 0 ? N : 1);
    // with every partner run given, Jaccard keys carry the row lengths
    // (the row field's spare bits) and no value array is kept
    if (sr == kJaccard && runs_given) cx.lenbits = 32 - cx.rowbits;
    cx.val = vb_out && cx.lenbits == 0 ? ar.get(size_t(N > 0 ? N : 1) * vb_out) : nullptr;

    if (N > 0) {
        // records (column, row, entry index) sorted by column; values are
        // gathered by entry index when the keys are packed
        uint32_t* ka = ar.get_t<uint32_t>(N);
        uint32_t* kb = ar.get_t<uint32_t>(N);
        uint32_t* ra = ar.get_t<uint32_t>(N);
        uint32_t* rb = ar.get_t<uint32_t>(N);
        // with no run table and no entry map the local sort needs the entries'
        // values only, so the passes carry them instead of the entry indices
        const int carried = runs_given && !run && !vsrc && (vb == 4 || vb == 8) && B.v &&
                                    local_bits(N, nbits_n) > 0
                                ? vb
                                : 0;
        const size_t eb_bytes = size_t(N) * size_t(carried ? carried : int(sizeof(uint32_t)));
        uint32_t* ea = static_cast<uint32_t*>(ar.get(eb_bytes));
        uint32_t* eb = static_cast<uint32_t*>(ar.get(eb_bytes));
        void* tmp = ar.get(radix_csr_tmp_bytes(N, nbits_n));
        // Jaccard keeps the row lengths in the row field's spare bits
        const int lenbits = sr == kJaccard ? 32 - cx.rowbits : 0;
        // with no directory a local sort writes the index itself (keys and
        // values at sorted positions, partner runs, the kept count)
        LocalPack pk;
        if (runs_given) {
            if (run) pk.run = *run;
            pk.key = cx.key;
            pk.val = cx.val;
            pk.vals_b = B.v;
            pk.rp_b = B.rp;
            pk.vbytes = vb;
            pk.jac = sr == kJaccard;
            pk.rowbits = cx.rowbits;
            pk.lenbits = lenbits;
            pk.drop_last = drop_last;
            pk.kept = &ctl->nkept;
            pk.ccount = ccount;
            pk.vsrc = vsrc;  // (ctl->nkept is zero: ctl is zeroed at the call's start)
            pk.carried = carried;
        }
        const int which = radix_sort_csr(B.ci, B.rp, B.m, cx.rowbits, lenbits, ka, kb, ra, rb, ea, eb, N, nbits_n, tmp,
                                         s, runs_given ? &pk : nullptr, hist1, trow1);
        check_launch();
        ar.release(tmp);
        if (counted) *counted = which < 0 && ccount;
        if (which >= 0) {
            void* ctmp = ar.get(colindex_tmp_bytes(N));
            build_colindex(which ? kb : ka, which ? rb : ra, which ? eb : ea, N, drop_last, vb, sr, B.v, B.rp, lenbits,
                           cx, ctmp, &ctl->nkept, run ? *run : RunTab(), s, vsrc);
            check_launch();
            ar.release(ctmp);
        }
        ar.release(ka);
        ar.release(kb);
        ar.release(ra);
        ar.release(rb);
        ar.release(ea);
        ar.release(eb);
    } else {
        void* ctmp = ar.get(colindex_tmp_bytes(0));
        build_colindex(nullptr, nullptr, nullptr, 0, drop_last, vb, sr, B.v, B.rp, 0, cx, ctmp, &ctl->nkept, RunTab(), s);
        check_launch();
        ar.release(ctmp);
    }
    return cx;
}

void zero_ctl(Ctl* ctl, hipStream_t s) { HIPCHK(hipMemsetAsync(ctl, 0, sizeof(Ctl), s)); }

spsyrk_status finish(spsyrk_status st) {
    if (st == SPSYRK_OK) g_detail.clear();
    return st;
}

// Rows per wavefront chunk of the light-row kernel (SPSYRK_ROWS_PER_CHUNK
// overrides it for tuning); a chunk splits into as many LDS batches as needed.
// A matrix of fewer rows than the device's wavefronts hold in chunks of
// kFusedRows takes shorter chunks (down to 8 rows), so that more wavefronts
// share it: tiny_uniform_f64 (4096 rows) 28 -> 17 us.
int rows_per_chunk(int64_t m) {
    if (const char* e = std::getenv("SPSYRK_ROWS_PER_CHUNK")) {
        const int v = std::atoi(e);
        if (v >= 1 && v <= kFusedRows) return v;
    }
    constexpr int64_t kWaves = 3072;  // wavefronts of the light kernel resident on the device
    int r = kFusedRows;
    while (r > 8 && m < int64_t(r) * kWaves) r /= 2;
    return r;
}

constexpr int64_t kDenseColumns = int64_t(1) << 28;  // dense column starts: at most 1 GiB

// What a lower product keeps for later products with new values on the same
// pattern: everything that depends on the pattern only (the column index and
// the entry behind each of its positions, partner runs, product counts, row
// classes, heavy rows' lengths and cursors, the output row pointers).
struct LowerPlan {
    int sr = 0;
    int64_t m = 0, n = 0, nnz = 0;
    bool empty = false;  // no products: every execution gives the empty result
    int64_t* rp = nullptr;  // copies of the pattern
    int32_t* ci = nullptr;
    ColIndex cx;
    uint32_t* vsrc = nullptr;  // entry of A behind every position of the index (nnz)
    RunTab run;
    uint32_t* rend = nullptr;  // run ends of the heavy rows' entries (nnz, with cursor)
    unsigned long long* prod = nullptr;
    int32_t* heavy_rows = nullptr;
    int64_t nheavy = 0;
    int64_t* heavy_nnz = nullptr;
    uint32_t* cursor = nullptr;
    Ctl* ctl = nullptr;
    int64_t* c_rp = nullptr;
    int64_t total = 0;
    int rows_per_chunk = 0;
    int64_t nchunks = 0;
};

// The buffers build_index takes for the column index of B in lower mode
// (every partner run given), allocated ahead with Arena::reserve: the keys,
// two buffers each of sorted keys, rows and entries, the values (none for
// Jaccard, whose keys carry the lengths) and the sort's workspace.
void reserve_index(const DevCsr& B, int sr, Arena& ar) {
    const int64_t N = B.nnz;
    if (N <= 0) return;
    const int nbits = bit_width_u64(B.n > 1 ? uint64_t(B.n - 1) : 0);
    ar.reserve(size_t(N) * sizeof(uint32_t), 7);
    const int vb = csc_value_bytes(sr);
    if (vb && sr != kJaccard) ar.reserve(size_t(N) * size_t(vb));
    ar.reserve(radix_csr_tmp_bytes(N, nbits));
}

// Largest output allocated at the staging slots' size before its exact size
// is known (columns and values).
constexpr size_t kEarlyOutputBytes = size_t(16) << 30;

// C_L = tril(A A^T) (lower, R = L) or L R^T: column index with the partner
// run of every entry, per-row product counts, row classes, exact lengths of
// the heavy rows, the light rows computed once into upper-bound staging slots
// with their exact lengths, row pointers, compaction of the light rows, heavy
// rows' values.  Off the diagonal the column index of R keeps every entry and
// the partner run of an entry of L in column k is the whole column k of R,
// read from dense column starts.

// checked: waits for the operands' validation flags and throws on a bad
// operand; called before the first kernel that reads their indices.
// hist1 (optional): the first radix pass's digit counts of the sorted operand
// (R), counted by its validation; vrows (optional, lower mode): the
// validation's table of tile rows of A
void syrk_fused(const DevCsr& L, const DevCsr& R, bool lower, int sr, Arena& ar, Ctl* ctl, hipStream_t s,
                spsyrk_csr_out* C, const std::function<void()>& checked, LowerPlan* plan = nullptr,
                uint32_t* hist1 = nullptr, const int64_t* vrows = nullptr) {
    const int64_t m = L.m;
    const int vbo = out_value_bytes(sr);
    unsigned long long* prod = ar.get_t<unsigned long long>(m);
    HIPCHK(hipMemsetAsync(prod, 0, size_t(m) * sizeof(unsigned long long), s));
    // partner runs, packed where the index's positions leave room for the lengths
    RunTab run;
    run.r4 = ar.get_t<uint32_t>(L.nnz);
    run.r8 = ar.get_t<uint2>(L.nnz);
    run.radix = run_radix(lower ? L.nnz : R.nnz);
    run.inv = 1.0 / double(run.radix);
    int32_t* heavy_rows = ar.get_t<int32_t>(m);
    int64_t* ub = ar.get_t<int64_t>(m + 1);
    // (classify_rows sets ub[m] = 0, and the light kernel row_cnt[m] = 0)
    void* ptmp = ar.get(row_products_tmp_bytes(L.nnz));
    ColIndex cx;
    if (lower) {
        HIPCHK(hipMemsetAsync(run.r4, 0, size_t(L.nnz) * sizeof(uint32_t), s));
        if (run.radix == 1) HIPCHK(hipMemsetAsync(run.r8, 0, size_t(L.nnz) * sizeof(uint2), s));
        uint32_t* vsrc = nullptr;
        if (plan) {
            vsrc = ar.get_t<uint32_t>(L.nnz);
            HIPCHK(hipMemsetAsync(vsrc, 0, size_t(L.nnz) * sizeof(uint32_t), s));
            plan->vsrc = vsrc;
        }
        reserve_index(L, sr, ar);
        checked();
        Phase ph(SPSYRK_PHASE_COLINDEX, s);
        cx = build_index(L, true, sr, ar, ctl, s, &run, true, nullptr, nullptr, vsrc, hist1, vrows);
        if (hist1) ar.release(hist1);
    } else {
        checked();
        Phase ph(SPSYRK_PHASE_COLINDEX, s);
        // column starts of R: from the counts the local sort writes, else by counting
        uint32_t* cptr = ar.get_t<uint32_t>(R.n + 1);
        HIPCHK(hipMemsetAsync(cptr, 0, size_t(R.n + 1) * sizeof(uint32_t), s));
        bool counted = false;
        cx = build_index(R, false, sr, ar, ctl, s, nullptr, false, cptr, &counted, nullptr, hist1);
        if (hist1) ar.release(hist1);
        void* ctmp = ar.get(scan_tmp_bytes(R.n + 1));
        if (counted)
            scan_u32(cptr, cptr, R.n + 1, nullptr, ctmp, s);
        else
            column_starts(R.ci, R.nnz, R.n, cptr, ctmp, s);
        offdiag_runs(L.ci, L.nnz, cptr, run, s);
        check_launch();
        ar.release(ctmp);
        ar.release(cptr);
    }
    {
        Phase ph(SPSYRK_PHASE_RUNS, s);
        row_products(L.rp, m, L.nnz, run, ptmp, prod, s, vrows);
        classify_rows(L.rp, prod, m, lower, heavy_rows, &ctl->heavy_count, &ctl->light_cap, &ctl->products, ub, s,
                      &ctl->maxlen);
    }
    check_launch();
    // the row classes go to the host; the scan of the staging slots needs
    // none of them and runs meanwhile
    ctl_fetch(ctl, s);
    int64_t* ubp = ub;
    void* stmp = ar.get(scan_tmp_bytes(m + 1));
    {
        Phase ph(SPSYRK_PHASE_SCAN, s);
        scan_i64(ub, ubp, m + 1, &ctl->total2, stmp, s);
    }
    int64_t* row_cnt = ar.get_t<int64_t>(m + 1);
    int64_t* c_rp = ar.get_t<int64_t>(m + 1, true);
    Ctl h = ctl_wait();
    ar.release(ptmp);
    const int64_t nheavy = h.heavy_count;
    const int64_t light_cap = int64_t(h.light_cap);
    HeavyArgs ha;
    int64_t* heavy_nnz = nullptr;
    if (nheavy > 1) {
        // the rows with the most products first, so that none starts last
        void* otmp = ar.get(heavy_order_tmp_bytes(nheavy));
        heavy_order(heavy_rows, nheavy, prod, otmp, s);
        check_launch();
        ar.release(otmp);
    }
    if (nheavy > 0) {
        heavy_nnz = ar.get_t<int64_t>(m);
        ha.m = m;
        ha.rp = L.rp;
        ha.ci = L.ci;
        ha.val = L.v;
        ha.cx = cx;
        ha.m_right = R.m;
        ha.rp_right = R.rp;
        ha.lower = lower;
        ha.sr = sr;
        ha.heavy_rows = heavy_rows;
        ha.heavy_count = &ctl->heavy_count;
        ha.heavy_max = nheavy;
        ha.row_nnz = heavy_nnz;
        ha.run = run;
        ha.runs_ready = true;
        ha.cursor = ar.get_t<uint32_t>(L.nnz);
        ha.rend = ar.get_t<uint32_t>(L.nnz);
        Phase ph(SPSYRK_PHASE_HEAVY_SYMBOLIC, s);
        heavy_symbolic(ha, &ctl->queue, s);
    }
    check_launch();
    // counts and Jaccard values of the light rows staged as one word per
    // output (column and packed value) where the words fit: the counts are
    // at most the light rows' lengths, the partners' lengths at most the
    // largest row's
    uint32_t pack_rr = 0, pack_r2 = 0;
    if (lower && (sr == kCount || sr == kJaccard) && pack_staging()) {
        const uint64_t lmax = h.maxlen;
        const uint64_t r1 = (lmax < uint64_t(kFusedEntries) ? lmax : uint64_t(kFusedEntries)) + 1, r2 = lmax + 1;
        const uint64_t rr = sr == kJaccard ? r1 * r2 : r1;
        if (rr < (uint64_t(1) << 17) && uint64_t(m) * rr <= (uint64_t(1) << 32)) {
            pack_rr = uint32_t(rr);
            pack_r2 = sr == kJaccard ? uint32_t(r2) : 0u;
        }
    }
    int32_t* s_ci = ar.get_t<int32_t>(light_cap > 0 ? light_cap : 1);
    void* s_val = ar.get(size_t(pack_rr || light_cap <= 0 ? 1 : light_cap) * vbo);

    FusedArgs fa;
    fa.m = m;
    fa.rp = L.rp;
    fa.ci = L.ci;
    fa.val = L.v;
    fa.cx = cx;
    fa.m_right = R.m;
    fa.rp_right = R.rp;
    fa.lower = lower;
    fa.sr = sr;
    fa.prod = prod;
    fa.run = run;
    fa.heavy_nnz = heavy_nnz;
    fa.ubp = ubp;
    fa.row_cnt = row_cnt;
    const int64_t nlight = m - nheavy;
    fa.rows_per_chunk = rows_per_chunk(m);
    fa.nchunks = (m + fa.rows_per_chunk - 1) / fa.rows_per_chunk;
    fa.chunk_counter = &ctl->chunk_counter;  // (zero: ctl is zeroed at the call's start)
    fa.c_ci = s_ci;
    fa.c_val = s_val;
    fa.pack_rr = pack_rr;
    fa.pack_r2 = pack_r2;
    {
        Phase ph(SPSYRK_PHASE_LIGHT_NUMERIC, s);
        light_fused(fa, s);
    }
    check_launch();
    {
        Phase ph(SPSYRK_PHASE_SCAN, s);
        scan_i64(row_cnt, c_rp, m + 1, &ctl->total, stmp, s);
    }
    heavy_sums(heavy_rows, nheavy, L.rp, c_rp, ctl->heavy_sums, s);  // (counters for the statistics)
    check_launch();
    // With every row light the staging slots bound the output: it is then
    // allocated at that size and compacted before the host reads its exact
    // size, so that the device does not wait for the host (up to a bound on
    // the extra memory; the slots exceed the output by the merged products).
    const bool early = nheavy == 0 && size_t(light_cap) * size_t(4 + vbo) <= kEarlyOutputBytes;
    int64_t total = 0;
    int32_t* c_ci = nullptr;
    void* c_val = nullptr;
    auto compact = [&]() {
        void* ctmp = ar.get(compact_tmp_bytes(light_cap));
        Phase ph(SPSYRK_PHASE_COMPACT, s);
        compact_rows(m, light_cap, ubp, row_cnt, c_rp, s_ci, s_val, vbo, ctmp, c_ci, c_val, s, pack_rr ? sr : 0,
                     pack_rr, pack_r2, L.rp);
    };
    if (early) {
        const int64_t cap = light_cap > 0 ? light_cap : 1;
        c_ci = ar.get_t<int32_t>(cap, true);
        c_val = ar.get(size_t(cap) * vbo, true);
        ctl_fetch(ctl, s);
        compact();
        check_launch();
        h = ctl_wait();
        total = h.total;
    } else {
        h = read_ctl(ctl, s);
        total = h.total;
        c_ci = ar.get_t<int32_t>(total > 0 ? total : 1, true);
        c_val = ar.get(size_t(total > 0 ? total : 1) * vbo, true);
        compact();
        check_launch();
    }
    if (nheavy > 0) {
        ha.c_rp = c_rp;
        ha.c_ci = c_ci;
        ha.c_val = c_val;
        {
            Phase ph(SPSYRK_PHASE_HEAVY_NUMERIC, s);
            heavy_numeric(ha, &ctl->queue, s);
        }
        check_launch();
    }
    C->nrows = m;
    C->ncols = R.m;
    C->nnz = total;
    C->row_ptr = c_rp;
    C->col_idx = c_ci;
    C->values = c_val;
    if (plan) {
        plan->cx = cx;
        plan->run.r8 = static_cast<uint2*>(ar.keep(run.r8));
        plan->run.r4 = static_cast<uint32_t*>(ar.keep(run.r4));
        plan->run.radix = run.radix;
        plan->run.inv = run.inv;
        plan->prod = static_cast<unsigned long long*>(ar.keep(prod));
        ar.keep(cx.key);
        if (cx.val) ar.keep(cx.val);
        ar.keep(plan->vsrc);
        plan->heavy_rows = static_cast<int32_t*>(ar.keep(heavy_rows));
        plan->nheavy = nheavy;
        if (nheavy > 0) {
            plan->heavy_nnz = static_cast<int64_t*>(ar.keep(heavy_nnz));
            plan->cursor = static_cast<uint32_t*>(ar.keep(ha.cursor));
            plan->rend = static_cast<uint32_t*>(ar.keep(ha.rend));
        }
        plan->ctl = static_cast<Ctl*>(ar.keep(ctl));
        plan->c_rp = ar.get_t<int64_t>(m + 1, true);
        HIPCHK(hipMemcpyAsync(plan->c_rp, c_rp, size_t(m + 1) * sizeof(int64_t), hipMemcpyDeviceToDevice, s));
        plan->total = total;
        plan->rows_per_chunk = fa.rows_per_chunk;
        plan->nchunks = fa.nchunks;
    }
    spsyrk_stats st{};
    st.nnz_out = total;
    st.csc_entries = h.nkept;
    st.heavy_rows = nheavy;
    st.light_rows = nlight;
    st.heavy_entries = int64_t(h.heavy_sums[0]);
    st.heavy_nnz_out = int64_t(h.heavy_sums[1]);
    st.products = int64_t(h.products);
    st.group_shift = cx.gs;
    st.row_bits = cx.rowbits;
    st.packed_staging = pack_rr != 0 ? 1 : 0;
    g_stats = st;
    g_stats_valid = true;
}

// C = tril(L R^T) (lower) or L R^T (offdiag), with R = L for lower.
void syrk(const DevCsr& L, const DevCsr& R, bool lower, int sr, Arena& ar, hipStream_t s, spsyrk_csr_out* C,
          LowerPlan* plan = nullptr) {
    Ctl* ctl = ar.get_t<Ctl>(1);
    zero_ctl(ctl, s);
    // on the single-pass path the validation of the operand whose columns
    // are sorted (R, which is L in lower mode) also counts the first radix
    // pass's digits
    const bool fused = (plan || !two_pass()) && (lower || R.n <= kDenseColumns);
    FirstHist fh;
    if (fused && R.nnz > 0 && L.m > 0 && L.nnz > 0) {
        radix_first_digit(R.nnz, bit_width_u64(R.n > 1 ? uint64_t(R.n - 1) : 0), &fh.shift, &fh.mask);
        fh.ntiles = (R.nnz + kRadixTile - 1) / kRadixTile;
        fh.hist = ar.get_t<uint32_t>(size_t(fh.ntiles) * 256);
    }
    // in lower mode the validation's table of tile rows of A serves the
    // first radix pass and the row products too
    void* vrows = fused && lower && L.nnz > 0 ? ar.get(validate_tmp_bytes(L.nnz)) : nullptr;
    {
        Phase ph(SPSYRK_PHASE_VALIDATE, s);
        validate_enqueue(L, false, ar, &ctl->err, s, lower && fh.hist ? &fh : nullptr, vrows);
        if (!lower) validate_enqueue(R, false, ar, &ctl->err2, s, fh.hist ? &fh : nullptr);
    }
    // The flags are read with one copy and checked before any kernel reads
    // the matrices' indices; the single-pass path first enqueues the
    // allocations and clears that depend on the sizes alone, so that the
    // host prepares them while the validation runs.
    ctl_fetch(ctl, s);
    const std::function<void()> checked = [&]() {
        const Ctl h = ctl_wait();
        check_valid(h.err, lower ? "A" : "Ai");
        if (!lower) check_valid(h.err2, "Aj");
    };

    const int64_t m = L.m;
    spsyrk_stats st{};
    if (m == 0 || L.nnz == 0 || R.nnz == 0) {
        checked();
        int64_t* c_rp = ar.get_t<int64_t>(m + 1, true);
        HIPCHK(hipMemsetAsync(c_rp, 0, size_t(m + 1) * sizeof(int64_t), s));
        C->nrows = m;
        C->ncols = R.m;
        C->row_ptr = c_rp;
        C->col_idx = ar.get_t<int32_t>(1, true);
        C->values = ar.get(4 * 2, true);
        C->nnz = 0;
        HIPCHK(hipStreamSynchronize(s));
        g_stats = st;
        g_stats_valid = true;
        if (plan) plan->empty = true;
        return;
    }

    // single pass over the light rows; off the diagonal when the right
    // operand's column starts fit a dense array (else the two-pass path)
    if (fused) {
        syrk_fused(L, R, lower, sr, ar, ctl, s, C, checked, plan, fh.hist, static_cast<const int64_t*>(vrows));
        return;
    }
    checked();
    int64_t* c_rp = ar.get_t<int64_t>(m + 1, true);
    ColIndex cx;
    {
        Phase ph(SPSYRK_PHASE_COLINDEX, s);
        cx = build_index(R, lower, sr, ar, ctl, s);
    }

    // symbolic
    int32_t* heavy_rows = ar.get_t<int32_t>(m);
    HIPCHK(hipMemsetAsync(c_rp + m, 0, sizeof(int64_t), s));
    LightArgs la;
    la.m = m;
    la.rp = L.rp;
    la.ci = L.ci;
    la.val = L.v;
    la.cx = cx;
    la.m_right = R.m;
    la.lower = lower;
    la.sr = sr;
    la.row_nnz = c_rp;
    la.heavy_rows = heavy_rows;
    la.heavy_count = &ctl->heavy_count;
    la.products = &ctl->products;
    {
        Phase ph(SPSYRK_PHASE_LIGHT_SYMBOLIC, s);
        light_symbolic(la, s);
    }
    check_launch();
    Ctl h = read_ctl(ctl, s);
    const int64_t nheavy = h.heavy_count;

    HeavyArgs ha;
    ha.m = m;
    ha.rp = L.rp;
    ha.ci = L.ci;
    ha.val = L.v;
    ha.cx = cx;
    ha.m_right = R.m;
    ha.rp_right = R.rp;
    ha.lower = lower;
    ha.sr = sr;
    ha.heavy_rows = heavy_rows;
    ha.heavy_count = &ctl->heavy_count;
    ha.heavy_max = nheavy;
    ha.products = &ctl->products;
    ha.row_nnz = c_rp;
    if (nheavy > 0) {
        ha.run.r8 = ar.get_t<uint2>(L.nnz);
        ha.cursor = ar.get_t<uint32_t>(L.nnz);
        ha.rend = ar.get_t<uint32_t>(L.nnz);
        {
            Phase ph(SPSYRK_PHASE_HEAVY_SYMBOLIC, s);
            heavy_symbolic(ha, &ctl->queue, s);
        }
        check_launch();
    }
    void* stmp = ar.get(scan_tmp_bytes(m + 1));
    {
        Phase ph(SPSYRK_PHASE_SCAN, s);
        scan_i64(c_rp, c_rp, m + 1, &ctl->total, stmp, s);
    }
    heavy_sums(heavy_rows, nheavy, L.rp, c_rp, ctl->heavy_sums, s);  // (counters for the statistics)
    check_launch();
    h = read_ctl(ctl, s);
    ar.release(stmp);
    const int64_t total = h.total;
    if (total >= (int64_t(1) << 62)) {
        set_detail("output size overflow");
        throw Fail{SPSYRK_ERR_OVERFLOW};
    }
    int32_t* c_ci = ar.get_t<int32_t>(total > 0 ? total : 1, true);
    void* c_val = ar.get(size_t(total > 0 ? total : 1) * out_value_bytes(sr), true);

    la.c_rp = c_rp;
    la.c_ci = c_ci;
    la.c_val = c_val;
    {
        Phase ph(SPSYRK_PHASE_LIGHT_NUMERIC, s);
        light_numeric(la, s);
    }
    check_launch();
    if (nheavy > 0) {
        ha.c_rp = c_rp;
        ha.c_ci = c_ci;
        ha.c_val = c_val;
        {
            Phase ph(SPSYRK_PHASE_HEAVY_NUMERIC, s);
            heavy_numeric(ha, &ctl->queue, s);
        }
        check_launch();
    }
    C->nrows = m;
    C->ncols = R.m;
    C->nnz = total;
    C->row_ptr = c_rp;
    C->col_idx = c_ci;
    C->values = c_val;

    st.nnz_out = total;
    st.csc_entries = h.nkept;
    st.heavy_rows = nheavy;
    st.light_rows = m - nheavy;
    st.heavy_entries = int64_t(h.heavy_sums[0]);
    st.heavy_nnz_out = int64_t(h.heavy_sums[1]);
    st.products = int64_t(h.products);
    st.group_shift = cx.gs;
    st.row_bits = cx.rowbits;
    g_stats = st;
    g_stats_valid = true;
}

// Strict-lower records per transpose slab: 2^31 (SPSYRK_MIRROR_SLAB, read at
// every call, lowers it to exercise the multi-slab path on small inputs).
int64_t mirror_slab_cap() {
    if (const char* e = std::getenv("SPSYRK_MIRROR_SLAB")) {
        const long long v = std::atoll(e);
        if (v >= 1 && v < (1LL << 31)) return int64_t(v);
    }
    return int64_t(1) << 31;
}

// columns [c0, c1) of the strict lower part, nrec of its entries, and the
// strict-lower entries in the columns before c0
struct Slab {
    int64_t c0, c1, nrec, before;
};

// Column slabs of at most cap strict-lower entries (a single column may hold
// more: it is a slab of its own) and at most wcap columns (wcap a multiple of
// the buckets' width), chosen from bucket histograms; a bucket over the cap
// is split by a finer histogram of its own columns.
std::vector<Slab> plan_slabs(const MirrorArgs& ma, int64_t cap, int64_t wcap, Arena& ar, hipStream_t s) {
    unsigned long long* hist = ar.get_t<unsigned long long>(kMirrorBins);
    std::vector<unsigned long long> h(kMirrorBins);
    std::vector<Slab> pieces;  // buckets (or single columns) in column order
    std::function<void(int64_t, int64_t)> refine = [&](int64_t lo, int64_t hi) {
        const int64_t w = hi - lo;
        int cb = 0;
        while (((w + (int64_t(1) << cb) - 1) >> cb) > kMirrorBins) ++cb;
        const int nb = int((w + (int64_t(1) << cb) - 1) >> cb);
        mirror_coarse_hist(ma, lo, cb, nb, hist, s);
        check_launch();
        HIPCHK(hipMemcpyAsync(h.data(), hist, size_t(nb) * sizeof(unsigned long long), hipMemcpyDeviceToHost, s));
        HIPCHK(hipStreamSynchronize(s));
        const std::vector<unsigned long long> hb(h.begin(), h.begin() + nb);
        for (int b = 0; b < nb; ++b) {
            const int64_t blo = lo + (int64_t(b) << cb);
            const int64_t bhi = std::min(hi, blo + (int64_t(1) << cb));
            if (int64_t(hb[size_t(b)]) > cap && bhi - blo > 1)
                refine(blo, bhi);
            else
                pieces.push_back({blo, bhi, int64_t(hb[size_t(b)]), 0});
        }
    };
    if (ma.m > 0) refine(0, ma.m);
    std::vector<Slab> out;
    Slab cur{0, 0, 0, 0};
    int64_t before = 0;
    for (const Slab& p : pieces) {
        if (cur.c1 > cur.c0 && (cur.nrec + p.nrec > cap || p.c1 - cur.c0 > wcap)) {
            out.push_back(cur);
            cur = {p.c0, p.c0, 0, before};
        }
        cur.c1 = p.c1;
        cur.nrec += p.nrec;
        before += p.nrec;
    }
    out.push_back(cur);
    ar.release(hist);
    return out;
}

void mirror(const DevCsr& L, int sr, Arena& ar, hipStream_t s, spsyrk_csr_out* C) {
    Ctl* ctl = ar.get_t<Ctl>(1);
    zero_ctl(ctl, s);
    {
        Phase ph(SPSYRK_PHASE_VALIDATE, s);
        validate(L, true, ar, ctl, s, "C_lower");
    }
    const int64_t m = L.m;
    const int vb = L.v ? out_value_bytes(sr) : 0;
    MirrorArgs ma;
    ma.m = m;
    ma.nnz = L.nnz;
    ma.rp = L.rp;
    ma.ci = L.ci;
    ma.val = L.v;
    ma.vbytes = vb;

    // The strict lower part is transposed in column slabs: records (column,
    // row, value) extracted row-major, sorted stably by column, each column's
    // record range read off the sorted keys, which gives the full row lengths
    // and starts of the slab's rows, and every record placed after the lower
    // part of its row.  The lower rows are copied once all starts are known.
    const int64_t cap = mirror_slab_cap();
    // Slabs of at most 2^16 columns sort in two 8-bit passes instead of
    // three: worth it when the records are many per row (each slab costs a
    // walk over every row's pointers).
    // (SPSYRK_MIRROR_NARROW=b, 1 <= b <= 16, read at every call: always
    // narrow, 2^b columns; 0: never)
    int64_t nwidth = kMirrorNarrow;
    const int64_t nslab16 = (m + kMirrorNarrow - 1) / kMirrorNarrow;
    bool narrow = nslab16 > 1 && L.nnz / 64 >= m * nslab16;
    if (const char* e = std::getenv("SPSYRK_MIRROR_NARROW")) {
        const int b = std::atoi(e);
        narrow = b >= 1 && b <= 16;
        if (narrow) nwidth = int64_t(1) << b;
    }
    const int64_t wcap = narrow ? nwidth : std::max<int64_t>(m, 1);
    // row of every tile start of the walks over C_L's entries
    int64_t* trow = ar.get_t<int64_t>(int64_t(mirror_tile_bytes(L.nnz) / sizeof(int64_t)));
    mirror_tile_rows(L.rp, m, trow, s);
    int64_t* row_cnt = ar.get_t<int64_t>(m + 1);
    int64_t* row_lo = ar.get_t<int64_t>(m > 0 ? m : 1);
    void* stmp = ar.get(scan_tmp_bytes(m + 1));
    std::vector<Slab> slabs;
    {
        Phase ph(SPSYRK_PHASE_MIRROR_COUNT, s);
        if (L.nnz <= cap && !narrow) {
            // one slab; its record count is the strict-lower count
            HIPCHK(hipMemsetAsync(row_cnt + m, 0, sizeof(int64_t), s));
            mirror_slab_counts(ma, 0, m, row_cnt, row_lo, s);
            scan_i64(row_cnt, row_cnt, m + 1, &ctl->total, stmp, s);
            check_launch();
            const Ctl h = read_ctl(ctl, s);
            slabs.push_back({0, m, h.total, 0});
        } else {
            slabs = plan_slabs(ma, cap, wcap, ar, s);
        }
    }
    int64_t nstrict = 0, rec_max = 0, w_max = 0;
    for (const Slab& sl : slabs) {
        nstrict += sl.nrec;
        rec_max = std::max(rec_max, sl.nrec);
        w_max = std::max(w_max, sl.c1 - sl.c0);
    }
    const int64_t total = L.nnz + nstrict;
    int64_t* f_rp = ar.get_t<int64_t>(m + 1, true);
    int32_t* f_ci = ar.get_t<int32_t>(total > 0 ? total : 1, true);
    void* f_val = vb ? ar.get(size_t(total > 0 ? total : 1) * vb, true) : nullptr;
    HIPCHK(hipMemsetAsync(f_rp, 0, sizeof(int64_t), s));  // m == 0: the only row start

    uint32_t* first = ar.get_t<uint32_t>(w_max > 0 ? w_max : 1);
    uint32_t* endc = ar.get_t<uint32_t>(w_max > 0 ? w_max : 1);
    uint32_t* ka = ar.get_t<uint32_t>(rec_max > 0 ? rec_max : 1);
    uint32_t* kb = ar.get_t<uint32_t>(rec_max > 0 ? rec_max : 1);
    uint32_t* ra = ar.get_t<uint32_t>(rec_max > 0 ? rec_max : 1);
    uint32_t* rb = ar.get_t<uint32_t>(rec_max > 0 ? rec_max : 1);
    void* va = vb ? ar.get(size_t(rec_max > 0 ? rec_max : 1) * vb) : nullptr;
    void* vbb = vb ? ar.get(size_t(rec_max > 0 ? rec_max : 1) * vb) : nullptr;
    void* rtmp = ar.get(radix_tmp_bytes(rec_max > 0 ? rec_max : 1));
    int64_t* strow = ar.get_t<int64_t>(int64_t(mirror_tile_bytes(rec_max) / sizeof(int64_t)));
    for (size_t k = 0; k < slabs.size(); ++k) {
        const Slab& sl = slabs[k];
        if (sl.c1 <= sl.c0) continue;
        Phase ph(SPSYRK_PHASE_MIRROR_TRANSPOSE, s);
        if (k > 0 || L.nnz > cap || narrow) {
            HIPCHK(hipMemsetAsync(row_cnt + m, 0, sizeof(int64_t), s));
            mirror_slab_counts(ma, sl.c0, sl.c1, row_cnt, row_lo, s);
            scan_i64(row_cnt, row_cnt, m + 1, &ctl->total, stmp, s);
            check_launch();
            if (read_ctl(ctl, s).total != sl.nrec) {  // the record buffers are sized from the histogram
                set_detail("mirror: slab record count disagrees with the column histogram");
                throw Fail{SPSYRK_ERR_HIP};
            }
        }
        const uint32_t* skey = ka;
        const uint32_t* srow = ra;
        const void* sval = va;
        const int nbits = bit_width_u64(sl.c1 - sl.c0 > 1 ? uint64_t(sl.c1 - sl.c0 - 1) : 0);
        // keys of at most 16 bits: the sort reads the records straight from
        // C_L and its last pass puts them into the full rows; wider keys go
        // through extracted records, passes and a placement
        const bool fused = nbits <= 16;
        if (sl.nrec > 0 && fused) {
            SlabIo io;
            io.ci = L.ci;
            io.val = vb ? L.v : nullptr;
            io.row_off = row_lo;
            io.c0 = sl.c0;
            io.rp = L.rp;
            io.before = sl.before;
            io.f_ci = f_ci;
            io.f_val = f_val;
            // (SPSYRK_SLAB_DIRECT=0, read at every call: the first pass reads
            // extracted records instead of C_L itself, about 4% slower on
            // R-MAT's transpose)
            const char* de = std::getenv("SPSYRK_SLAB_DIRECT");
            const bool direct = !(de && de[0] == '0');
            if (direct)
                mirror_slab_offsets(row_lo, row_cnt, m, s);
            else
                mirror_slab_extract(ma, sl.c0, sl.nrec, row_cnt, row_lo, strow, ka, ra, va, s);
            skey = slab_sort_place(io, vb, sl.nrec, nbits, row_cnt, m, !direct, ka, kb, ra, rb, va, vbb, rtmp, s);
        } else if (sl.nrec > 0) {
            mirror_slab_extract(ma, sl.c0, sl.nrec, row_cnt, row_lo, strow, ka, ra, va, s);
            if (radix_sort(ka, kb, ra, rb, va, vbb, vb, sl.nrec, nbits, rtmp, s)) {
                skey = kb;
                srow = rb;
                sval = vbb;
            }
        }
        // row_cnt is free again: full lengths of the slab's rows
        mirror_slab_columns(ma, sl.c0, sl.c1, skey, sl.nrec, first, endc, row_cnt, sl.before, f_rp, stmp, s);
        if (!fused) mirror_slab_place(ma, sl.c0, sl.nrec, skey, srow, sval, first, f_rp, f_ci, f_val, s);
        check_launch();
    }
    {
        Phase ph(SPSYRK_PHASE_MIRROR_COPY, s);
        mirror_copy_lower(ma, 0, L.nnz, trow, f_rp, f_ci, f_val, s);
    }
    check_launch();
    HIPCHK(hipStreamSynchronize(s));
    C->nrows = m;
    C->ncols = m;
    C->nnz = total;
    C->row_ptr = f_rp;
    C->col_idx = f_ci;
    C->values = f_val;
    spsyrk_stats st{};
    st.nnz_out = total;
    g_stats = st;
    g_stats_valid = true;
}

// one device int64 read back to the host (one synchronisation)
int64_t read_i64(const int64_t* d, hipStream_t s) {
    struct Pinned {
        int64_t* h = nullptr;
        Pinned() {
            if (hipHostMalloc(reinterpret_cast<void**>(&h), sizeof(int64_t), hipHostMallocDefault) != hipSuccess)
                h = nullptr;
        }
        ~Pinned() {
            if (h) (void)hipHostFree(h);
        }
    };
    thread_local Pinned pin;
    if (!pin.h) {
        set_detail("pinned host buffer unavailable");
        throw Fail{SPSYRK_ERR_HIP};
    }
    HIPCHK(hipMemcpyAsync(pin.h, d, sizeof(int64_t), hipMemcpyDeviceToHost, s));
    HIPCHK(hipStreamSynchronize(s));
    return *pin.h;
}

// Half of an off-diagonal block (Algorithm 3): the top rows [0, floor(m_i/2))
// of A_i A_j^T, or its right columns [floor(m_j/2), m_j).  Both are the
// off-diagonal product of a row range of one operand; the right half's
// column ids are shifted back to the block's numbering.
void offdiag_half(const DevCsr& L, const DevCsr& R, int half, int sr, Arena& ar, hipStream_t s, spsyrk_csr_out* C) {
    const int vb = (sr == kF64) ? 8 : (sr == kF32 ? 4 : 0);
    if (half == SPSYRK_HALF_TOP) {
        DevCsr T = L;
        T.m = L.m / 2;
        // (the row pointer prefix is the top rows' own; their nnz is rp[m/2])
        T.nnz = read_i64(L.rp + T.m, s);
        if (T.nnz < 0 || T.nnz > L.nnz) {
            set_detail("Ai is not canonical CSR (row_ptr[%lld] = %lld)", (long long)T.m, (long long)T.nnz);
            throw Fail{SPSYRK_ERR_NOT_CANONICAL};
        }
        syrk(T, R, false, sr, ar, s, C);
        return;
    }
    const int64_t c0 = R.m / 2;
    const int64_t e0 = read_i64(R.rp + c0, s);
    if (e0 < 0 || e0 > R.nnz) {
        set_detail("Aj is not canonical CSR (row_ptr[%lld] = %lld)", (long long)c0, (long long)e0);
        throw Fail{SPSYRK_ERR_NOT_CANONICAL};
    }
    DevCsr B = R;
    B.m = R.m - c0;
    B.nnz = R.nnz - e0;
    int64_t* rp = ar.get_t<int64_t>(B.m + 1);
    rebase_rows(R.rp, c0, B.m, rp, s);
    check_launch();
    B.rp = rp;
    B.ci = R.ci + e0;
    B.v = R.v ? static_cast<const char*>(R.v) + e0 * vb : nullptr;
    syrk(L, B, false, sr, ar, s, C);
    shift_columns(C->col_idx, C->nnz, int32_t(c0), s);
    check_launch();
    C->ncols = R.m;
}

// A lower product on a planned pattern with new values: the values of the
// column index gathered from the new values, then the light rows written
// straight into their final places (their lengths are known) and the heavy
// rows; no sort, no symbolic pass, no staging, no compaction, no host wait.
void lower_execute(const LowerPlan& P, const void* vals, Arena& ar, hipStream_t s, spsyrk_csr_out* C) {
    const int64_t m = P.m;
    const int vbo = out_value_bytes(P.sr);
    int64_t* c_rp = ar.get_t<int64_t>(m + 1, true);
    const int64_t total = P.empty ? 0 : P.total;
    int32_t* c_ci = ar.get_t<int32_t>(total > 0 ? total : 1, true);
    void* c_val = ar.get(size_t(total > 0 ? total : 1) * vbo, true);
    C->nrows = m;
    C->ncols = m;
    C->nnz = total;
    C->row_ptr = c_rp;
    C->col_idx = c_ci;
    C->values = c_val;
    if (P.empty) {
        HIPCHK(hipMemsetAsync(c_rp, 0, size_t(m + 1) * sizeof(int64_t), s));
        return;
    }
    HIPCHK(hipMemcpyAsync(c_rp, P.c_rp, size_t(m + 1) * sizeof(int64_t), hipMemcpyDeviceToDevice, s));
    const int vb = (P.sr == kF64) ? 8 : (P.sr == kF32 ? 4 : 0);
    if (vb) {
        gather_values(P.cx.val, vals, P.vsrc, P.nnz, vb, s);
        check_launch();
    }
    int64_t* row_cnt = ar.get_t<int64_t>(m + 1);
    FusedArgs fa;
    fa.m = m;
    fa.rp = P.rp;
    fa.ci = P.ci;
    fa.val = vals;
    fa.cx = P.cx;
    fa.m_right = m;
    fa.rp_right = P.rp;
    fa.lower = true;
    fa.sr = P.sr;
    fa.prod = P.prod;
    fa.run = P.run;
    fa.heavy_nnz = P.heavy_nnz;
    fa.ubp = P.c_rp;  // the final row starts: the light rows land in place
    fa.row_cnt = row_cnt;
    fa.rows_per_chunk = P.rows_per_chunk;
    fa.nchunks = P.nchunks;
    HIPCHK(hipMemsetAsync(&P.ctl->chunk_counter, 0, sizeof(P.ctl->chunk_counter), s));
    fa.chunk_counter = &P.ctl->chunk_counter;
    fa.c_ci = c_ci;
    fa.c_val = c_val;
    {
        Phase ph(SPSYRK_PHASE_LIGHT_NUMERIC, s);
        light_fused(fa, s);
    }
    check_launch();
    if (P.nheavy > 0) {
        HeavyArgs ha;
        ha.m = m;
        ha.rp = P.rp;
        ha.ci = P.ci;
        ha.val = vals;
        ha.cx = P.cx;
        ha.m_right = m;
        ha.rp_right = P.rp;
        ha.lower = true;
        ha.sr = P.sr;
        ha.heavy_rows = P.heavy_rows;
        ha.heavy_count = &P.ctl->heavy_count;
        ha.heavy_max = P.nheavy;
        ha.row_nnz = P.heavy_nnz;
        ha.run = P.run;
        ha.runs_ready = true;
        ha.cursor = P.cursor;
        ha.rend = P.rend;
        ha.c_rp = c_rp;
        ha.c_ci = c_ci;
        ha.c_val = c_val;
        Phase ph(SPSYRK_PHASE_HEAVY_NUMERIC, s);
        heavy_numeric(ha, &P.ctl->queue, s);
    }
    check_launch();
    ar.release(row_cnt);
}

template <typename F>
spsyrk_status guarded(spsyrk_csr_out* C, const spsyrk_allocator* al, void* stream, F body) {
    g_stats_valid = false;
    if (!C) {
        set_detail("output struct is null");
        return SPSYRK_ERR_INVALID_ARG;
    }
    std::memset(C, 0, sizeof(*C));
    hipStream_t s = static_cast<hipStream_t>(stream);
    Arena ar(al, s);
    try {
        body(ar, s);
        ar.keep_outputs();
    } catch (const Fail& f) {
        ar.release_all();
        std::memset(C, 0, sizeof(*C));
        if (ar.touched()) (void)hipStreamSynchronize(s);
        return f.st;
    } catch (...) {
        ar.release_all();
        std::memset(C, 0, sizeof(*C));
        set_detail("unexpected host exception");
        return SPSYRK_ERR_HIP;
    }
    ar.release_all();
    return finish(SPSYRK_OK);
}

}  // namespace

// ---- scratch of the allocation-free product from a stored lower part
// (spsyrk_symm_noalloc): one array per device, held until the process ends.
// Its name is a host-side stand-in in host code; kernels get the device
// address that hipGetSymbolAddress returns for the current device.
constexpr size_t kScratchBytes = size_t(128) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of the current device's scratch, looked up once per
// device with that device current.
void* scratch_ptr() {
    int dev = 0;
    HIPCHK(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) {
        set_detail("device %d is beyond the %d devices the scratch table covers", dev, kMaxDevices);
        throw Fail{SPSYRK_ERR_HIP};
    }
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        HIPCHK(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p) {
            set_detail("hipGetSymbolAddress returned a null scratch address");
            throw Fail{SPSYRK_ERR_HIP};
        }
        g_scratch_ptr[dev] = p;
    }
    return g_scratch_ptr[dev];
}

// scratch layout: the validation word in the first 256 bytes, then the
// validation tile table, reused afterwards by the product's workspace
size_t symm_noalloc_bytes(int64_t m, int64_t k, int64_t nnz) {
    const size_t v = (validate_tmp_bytes(nnz) + 255) & ~size_t(255);
    const size_t w = symm_tmp_bytes(m, k, nnz, kSymmAtomics);
    return 256 + (v > w ? v : w);
}

}  // namespace

spsyrk::PhaseTimer::PhaseTimer(int phase, hipStream_t s) : s_(s), phase_(phase) {
    if (!g_timing || phase < 0 || phase >= 32 || !((g_phase_mask >> phase) & 1u)) return;
    a_ = pooled_event();
    b_ = pooled_event();
    if (!a_ || !b_ || hipEventRecord(a_, s_) != hipSuccess) {
        pool_event(a_);
        pool_event(b_);
        return;
    }
    on_ = true;
}

spsyrk::PhaseTimer::~PhaseTimer() {
    if (!on_) return;
    if (hipEventRecord(b_, s_) == hipSuccess) {
        g_marks.push_back(PhaseMark{phase_, a_, b_});
    } else {
        pool_event(a_);
        pool_event(b_);
    }
}

// the opaque plan handle of the C interface
struct spsyrk_plan_s {
    LowerPlan p;
    spsyrk_allocator al{};
    bool has_al = false;
    int device = 0;           // the device the buffers live on
    std::vector<void*> bufs;  // device buffers owned by the plan
};

namespace spsyrk {
namespace dbg {
// the debug build's per-unit readers, filled by static initialisers at load
std::vector<Reader>& readers() {
    static std::vector<Reader> v;
    return v;
}
void add_reader(Reader r) { readers().push_back(r); }
}  // namespace dbg
}  // namespace spsyrk

extern "C" {

spsyrk_status spsyrk_lower(const spsyrk_csr* A, spsyrk_semiring sr, const spsyrk_allocator* al, void* hip_stream,
                           spsyrk_csr_out* C) {
    return guarded(C, al, hip_stream, [&](Arena& ar, hipStream_t s) {
        check_semiring(int(sr));
        check_input(A, int(sr), true, "A");
        const DevCsr d = dev(A);
        syrk(d, d, true, int(sr), ar, s, C);
    });
}

spsyrk_status spsyrk_offdiag(const spsyrk_csr* Ai, const spsyrk_csr* Aj, spsyrk_semiring sr,
                             const spsyrk_allocator* al, void* hip_stream, spsyrk_csr_out* C) {
    return guarded(C, al, hip_stream, [&](Arena& ar, hipStream_t s) {
        check_semiring(int(sr));
        check_input(Ai, int(sr), true, "Ai");
        check_input(Aj, int(sr), true, "Aj");
        if (Ai->ncols != Aj->ncols) {
            set_detail("Ai has %lld columns, Aj has %lld", (long long)Ai->ncols, (long long)Aj->ncols);
            throw Fail{SPSYRK_ERR_INVALID_ARG};
        }
        syrk(dev(Ai), dev(Aj), false, int(sr), ar, s, C);
    });
}

spsyrk_status spsyrk_offdiag_half(const spsyrk_csr* Ai, const spsyrk_csr* Aj, spsyrk_half half,
                                  spsyrk_semiring sr, const spsyrk_allocator* al, void* hip_stream,
                                  spsyrk_csr_out* C) {
    return guarded(C, al, hip_stream, [&](Arena& ar, hipStream_t s) {
        check_semiring(int(sr));
        check_input(Ai, int(sr), true, "Ai");
        check_input(Aj, int(sr), true, "Aj");
        if (Ai->ncols != Aj->ncols) {
            set_detail("Ai has %lld columns, Aj has %lld", (long long)Ai->ncols, (long long)Aj->ncols);
            throw Fail{SPSYRK_ERR_INVALID_ARG};
        }
        if (half != SPSYRK_HALF_TOP && half != SPSYRK_HALF_RIGHT) {
            set_detail("unknown half %d", int(half));
            throw Fail{SPSYRK_ERR_INVALID_ARG};
        }
        offdiag_half(dev(Ai), dev(Aj), int(half), int(sr), ar, s, C);
    });
}

spsyrk_status spsyrk_symm(const spsyrk_csr* C_lower, spsyrk_semiring sr, int64_t k, const void* X, int64_t ldx,
                          void* Y, int64_t ldy, const spsyrk_allocator* al, void* hip_stream) {
    spsyrk_csr_out unused;
    return guarded(&unused, al, hip_stream, [&](Arena& ar, hipStream_t s) {
        check_semiring(int(sr));
        check_input(C_lower, int(sr), false, "C_lower", int64_t(1) << 62);
        if (C_lower->nrows != C_lower->ncols) {
            set_detail("C_lower must be square (%lld x %lld)", (long long)C_lower->nrows,
                       (long long)C_lower->ncols);
            throw Fail{SPSYRK_ERR_INVALID_ARG};
        }
        if (k < 0 || ldx < k || ldy < k) {
            set_detail("need 0 <= k <= ldx, ldy (k %lld, ldx %lld, ldy %lld)", (long long)k, (long long)ldx,
                       (long long)ldy);
            throw Fail{SPSYRK_ERR_INVALID_ARG};
        }
        const int64_t m = C_lower->nrows;
        if (m == 0 || k == 0) return;
        if (!X || !Y || (C_lower->nnz > 0 && !C_lower->values)) {
            set_detail("X, Y and the values of C_lower are required");
            throw Fail{SPSYRK_ERR_INVALID_ARG};
        }
        const DevCsr c = dev(C_lower);
        {
            Ctl* ctl = ar.get_t<Ctl>(1);
            zero_ctl(ctl, s);
            validate(c, true, ar, ctl, s, "C_lower");
        }
        const int mode = symm_mode(m, k, c.nnz);
        void* tmp = ar.get(symm_tmp_bytes(m, k, c.nnz, mode));
        symm_product(c, int(sr), X, ldx, k, Y, ldy, tmp, mode, s);
        check_launch();
        HIPCHK(hipStreamSynchronize(s));
    });
}

spsyrk_status spsyrk_symm_noalloc(const spsyrk_csr* C_lower, spsyrk_semiring sr, int64_t k, const void* X,
                                  int64_t ldx, void* Y, int64_t ldy, void* hip_stream) {
    g_stats_valid = false;
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    try {
        check_semiring(int(sr));
        check_input(C_lower, int(sr), false, "C_lower", int64_t(1) << 62);
        if (C_lower->nrows != C_lower->ncols) {
            set_detail("C_lower must be square (%lld x %lld)", (long long)C_lower->nrows,
                       (long long)C_lower->ncols);
            throw Fail{SPSYRK_ERR_INVALID_ARG};
        }
        if (k < 0 || ldx < k || ldy < k) {
            set_detail("need 0 <= k <= ldx, ldy (k %lld, ldx %lld, ldy %lld)", (long long)k, (long long)ldx,
                       (long long)ldy);
            throw Fail{SPSYRK_ERR_INVALID_ARG};
        }
        const int64_t m = C_lower->nrows;
        if (m == 0 || k == 0) return finish(SPSYRK_OK);
        if (!X || !Y || (C_lower->nnz > 0 && !C_lower->values)) {
            set_detail("X, Y and the values of C_lower are required");
            throw Fail{SPSYRK_ERR_INVALID_ARG};
        }
        const DevCsr c = dev(C_lower);
        const size_t need = symm_noalloc_bytes(m, k, c.nnz);
        if (need > kScratchBytes) {
            set_detail("needs %zu bytes of scratch, the allocation-free call holds %zu (m k = %lld)", need,
                       kScratchBytes, (long long)(m * k));
            throw Fail{SPSYRK_ERR_TOO_LARGE};
        }
        char* base = static_cast<char*>(scratch_ptr());
        uint32_t* err = reinterpret_cast<uint32_t*>(base);
        fill_u32(err, 1, 0u, s);
        validate_csr(c, true, err, base + 256, s);
        check_launch();
        uint32_t herr = 0;
        HIPCHK(hipMemcpyAsync(&herr, err, sizeof(herr), hipMemcpyDeviceToHost, s));
        HIPCHK(hipStreamSynchronize(s));
        if (herr) {
            set_detail("C_lower is not canonical CSR (flags 0x%x)", herr);
            throw Fail{SPSYRK_ERR_NOT_CANONICAL};
        }
        symm_product(c, int(sr), X, ldx, k, Y, ldy, base + 256, kSymmAtomics, s);
        check_launch();
        HIPCHK(hipStreamSynchronize(s));
    } catch (const Fail& f) {
        return f.st;
    } catch (...) {
        set_detail("unexpected host exception");
        return SPSYRK_ERR_HIP;
    }
    return finish(SPSYRK_OK);
}

spsyrk_status spsyrk_lower_accumulate(const spsyrk_csr* C_prev, const spsyrk_csr* A_s, spsyrk_semiring sr,
                                      const spsyrk_allocator* al, void* hip_stream, spsyrk_csr_out* C) {
    return guarded(C, al, hip_stream, [&](Arena& ar, hipStream_t s) {
        check_semiring(int(sr));
        if (sr == SPSYRK_COUNT_I32_JACCARD_F32) {
            set_detail("Jaccard values do not add across stages; accumulate overlap counts (COUNT_I32)");
            throw Fail{SPSYRK_ERR_INVALID_ARG};
        }
        check_input(C_prev, int(sr), false, "C_prev", int64_t(1) << 62);
        check_input(A_s, int(sr), true, "A_s");
        if (C_prev->nrows != C_prev->ncols || C_prev->nrows != A_s->nrows) {
            set_detail("C_prev must be m x m with m = A_s rows (%lld x %lld, %lld)", (long long)C_prev->nrows,
                       (long long)C_prev->ncols, (long long)A_s->nrows);
            throw Fail{SPSYRK_ERR_INVALID_ARG};
        }
        if (C_prev->nnz > 0 && !C_prev->values) {
            set_detail("C_prev values are required");
            throw Fail{SPSYRK_ERR_INVALID_ARG};
        }
        const int64_t m = A_s->nrows;
        const DevCsr P = dev(C_prev);
        {
            Ctl* ctl = ar.get_t<Ctl>(1);
            zero_ctl(ctl, s);
            validate(P, true, ar, ctl, s, "C_prev");
        }
        // this stage's lower part, an intermediate result
        spsyrk_csr_out t{};
        syrk(dev(A_s), dev(A_s), true, int(sr), ar, s, &t);
        DevCsr T;
        T.m = m;
        T.n = m;
        T.nnz = t.nnz;
        T.rp = t.row_ptr;
        T.ci = t.col_idx;
        T.v = t.values;
        // union of the two patterns, in chunks of rows and windows of long
        // rows: counts, row pointers, merge
        int64_t* fl = ar.get_t<int64_t>(m + 1);
        void* stmp = ar.get(scan_tmp_bytes(m + 1));
        merge_item_flags(m, P, T, fl, stmp, s);
        check_launch();
        const int64_t items = m > 0 ? read_i64(fl + m, s) : 0;
        int64_t* crow = ar.get_t<int64_t>(items + 1);
        int32_t* cwin = ar.get_t<int32_t>(items > 0 ? items : 1);
        int64_t* wsum = ar.get_t<int64_t>(items > 0 ? items : 1);
        merge_item_table(m, P, T, fl, crow, cwin, s);
        check_launch();
        int64_t* cnt = fl;  // the item counts are spent (same stream)
        HIPCHK(hipMemsetAsync(cnt, 0, sizeof(int64_t) * size_t(m + 1), s));
        merge_lower(false, int(sr), items, crow, cwin, P, T, cnt, wsum, nullptr, nullptr, nullptr, s);
        check_launch();
        int64_t* c_rp = ar.get_t<int64_t>(m + 1, true);
        scan_i64(cnt, c_rp, m + 1, nullptr, stmp, s);
        check_launch();
        ar.release(stmp);
        if (items > 0) {
            void* wtmp = ar.get(scan_tmp_bytes(items));
            scan_i64(wsum, wsum, items, nullptr, wtmp, s);
            check_launch();
            ar.release(wtmp);
        }
        const int64_t total = m > 0 ? read_i64(c_rp + m, s) : 0;
        const int vb = out_value_bytes(int(sr));
        int32_t* c_ci = ar.get_t<int32_t>(total > 0 ? total : 1, true);
        void* c_val = ar.get(size_t(total > 0 ? total : 1) * vb, true);
        merge_lower(true, int(sr), items, crow, cwin, P, T, nullptr, wsum, c_rp, c_ci, c_val, s);
        check_launch();
        HIPCHK(hipStreamSynchronize(s));
        ar.release(wsum);
        ar.release(cwin);
        ar.release(crow);
        ar.release(fl);
        ar.release_output(t.row_ptr);
        ar.release_output(t.col_idx);
        ar.release_output(t.values);
        C->nrows = m;
        C->ncols = m;
        C->nnz = total;
        C->row_ptr = c_rp;
        C->col_idx = c_ci;
        C->values = c_val;
    });
}

spsyrk_status spsyrk_lower_plan(const spsyrk_csr* A, spsyrk_semiring sr, const spsyrk_allocator* al,
                                void* hip_stream, spsyrk_plan** plan, spsyrk_csr_out* C) {
    if (!plan) {
        set_detail("plan is null");
        return SPSYRK_ERR_INVALID_ARG;
    }
    *plan = nullptr;
    spsyrk_plan* made = nullptr;
    const spsyrk_status st = guarded(C, al, hip_stream, [&](Arena& ar, hipStream_t s) {
        check_semiring(int(sr));
        check_input(A, int(sr), true, "A");
        const DevCsr d = dev(A);
        LowerPlan lp;
        syrk(d, d, true, int(sr), ar, s, C, &lp);
        lp.sr = int(sr);
        lp.m = d.m;
        lp.n = d.n;
        lp.nnz = d.nnz;
        lp.rp = ar.get_t<int64_t>(d.m + 1, true);
        HIPCHK(hipMemcpyAsync(lp.rp, d.rp, size_t(d.m + 1) * sizeof(int64_t), hipMemcpyDeviceToDevice, s));
        lp.ci = ar.get_t<int32_t>(d.nnz > 0 ? d.nnz : 1, true);
        if (d.nnz > 0)
            HIPCHK(hipMemcpyAsync(lp.ci, d.ci, size_t(d.nnz) * sizeof(int32_t), hipMemcpyDeviceToDevice, s));
        HIPCHK(hipStreamSynchronize(s));
        int device = 0;
        HIPCHK(hipGetDevice(&device));
        auto* h = new spsyrk_plan_s;
        h->p = lp;
        h->device = device;
        if (al) {
            h->al = *al;
            h->has_al = true;
        }
        for (void* q : {static_cast<void*>(lp.rp), static_cast<void*>(lp.ci), static_cast<void*>(lp.run.r8),
                        static_cast<void*>(lp.run.r4), static_cast<void*>(lp.rend),
                        static_cast<void*>(lp.prod), static_cast<void*>(lp.cx.key), lp.cx.val,
                        static_cast<void*>(lp.vsrc), static_cast<void*>(lp.heavy_rows),
                        static_cast<void*>(lp.heavy_nnz), static_cast<void*>(lp.cursor),
                        static_cast<void*>(lp.ctl), static_cast<void*>(lp.c_rp)})
            if (q) h->bufs.push_back(q);
        made = h;
    });
    if (st == SPSYRK_OK) *plan = made;
    return st;
}

spsyrk_status spsyrk_lower_execute(spsyrk_plan* plan, const void* values, const spsyrk_allocator* al,
                                   void* hip_stream, spsyrk_csr_out* C) {
    return guarded(C, al, hip_stream, [&](Arena& ar, hipStream_t s) {
        if (!plan) {
            set_detail("plan is null");
            throw Fail{SPSYRK_ERR_INVALID_ARG};
        }
        const LowerPlan& P = plan->p;
        if ((P.sr == kF64 || P.sr == kF32) && P.nnz > 0 && !values) {
            set_detail("values are required for plus-times semirings");
            throw Fail{SPSYRK_ERR_INVALID_ARG};
        }
        lower_execute(P, values, ar, s, C);
        spsyrk_stats st{};
        st.nnz_out = C->nnz;
        st.heavy_rows = P.nheavy;
        st.light_rows = P.m - P.nheavy;
        g_stats = st;
        g_stats_valid = true;
    });
}

spsyrk_status spsyrk_plan_destroy(spsyrk_plan* plan) {
    if (!plan) return SPSYRK_OK;
    if (plan->has_al) {
        if (plan->al.free)
            for (void* q : plan->bufs) plan->al.free(plan->al.ctx, q);
    } else {
        // the buffers came from hipMallocAsync: stream-ordered frees once the
        // device is idle, then a wait so that they are released on return
        int cur = 0;
        (void)hipGetDevice(&cur);
        (void)hipSetDevice(plan->device);
        (void)hipDeviceSynchronize();
        for (void* q : plan->bufs) (void)hipFreeAsync(q, nullptr);
        (void)hipStreamSynchronize(nullptr);
        (void)hipSetDevice(cur);
    }
    delete plan;
    return SPSYRK_OK;
}

spsyrk_status spsyrk_mirror(const spsyrk_csr* C_lower, spsyrk_semiring sr, const spsyrk_allocator* al,
                            void* hip_stream, spsyrk_csr_out* C_full) {
    return guarded(C_full, al, hip_stream, [&](Arena& ar, hipStream_t s) {
        check_semiring(int(sr));
        check_input(C_lower, int(sr), false, "C_lower", int64_t(1) << 62);
        if (C_lower->nrows != C_lower->ncols) {
            set_detail("C_lower must be square (%lld x %lld)", (long long)C_lower->nrows,
                       (long long)C_lower->ncols);
            throw Fail{SPSYRK_ERR_INVALID_ARG};
        }
        mirror(dev(C_lower), int(sr), ar, s, C_full);
    });
}

const char* spsyrk_status_string(spsyrk_status s) {
    switch (s) {
        case SPSYRK_OK: return "ok";
        case SPSYRK_ERR_INVALID_ARG: return "invalid argument";
        case SPSYRK_ERR_NOT_CANONICAL: return "input is not canonical CSR";
        case SPSYRK_ERR_SHAPE: return "shape out of range";
        case SPSYRK_ERR_OOM: return "out of device memory";
        case SPSYRK_ERR_OVERFLOW: return "count overflow";
        case SPSYRK_ERR_HIP: return "HIP runtime error";
        case SPSYRK_ERR_TOO_LARGE: return "operands exceed the fixed scratch of the allocation-free call";
    }
    return "unknown status";
}

const char* spsyrk_last_error_detail(void) { return g_detail.c_str(); }

int spsyrk_debug_build(void) {
#if defined(SPSYRK_DEBUG) && SPSYRK_DEBUG
    return 1;
#else
    return 0;
#endif
}

spsyrk_status spsyrk_debug_flags(uint32_t* flags) {
    if (!flags) {
        set_detail("spsyrk_debug_flags: flags is NULL");
        return SPSYRK_ERR_INVALID_ARG;
    }
    *flags = 0;
    const hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) {
        set_detail("hipDeviceSynchronize: %s", hipGetErrorString(e));
        return SPSYRK_ERR_HIP;
    }
    uint32_t f = 0;
    for (spsyrk::dbg::Reader r : spsyrk::dbg::readers()) f |= r();
    *flags = f;
    return SPSYRK_OK;
}

spsyrk_status spsyrk_last_stats(spsyrk_stats* out) {
    if (!out) return SPSYRK_ERR_INVALID_ARG;
    if (!g_stats_valid) {
        std::memset(out, 0, sizeof(*out));
        return SPSYRK_ERR_INVALID_ARG;
    }
    *out = g_stats;
    return SPSYRK_OK;
}

int spsyrk_abi_version(void) { return SPSYRK_ABI_VERSION; }

spsyrk_status spsyrk_timing_begin(void) { return spsyrk_timing_begin_phases(0xffffffffu); }

spsyrk_status spsyrk_timing_begin_phases(uint32_t mask) {
    for (auto& mk : g_marks) {
        pool_event(mk.a);
        pool_event(mk.b);
    }
    g_marks.clear();
    // enough events for a few calls' phases, created now rather than inside them
    while (g_event_pool.size() < 64) {
        hipEvent_t e = nullptr;
        if (hipEventCreate(&e) != hipSuccess) break;
        g_event_pool.push_back(e);
    }
    g_phase_mask = mask;
    g_timing = true;
    return SPSYRK_OK;
}

spsyrk_status spsyrk_timing_end(spsyrk_phase_times* out) {
    g_timing = false;
    spsyrk_status st = SPSYRK_OK;
    if (out) std::memset(out, 0, sizeof(*out));
    for (auto& mk : g_marks) {
        float ms = 0.f;
        if (hipEventSynchronize(mk.b) != hipSuccess || hipEventElapsedTime(&ms, mk.a, mk.b) != hipSuccess) {
            set_detail("phase event query failed");
            st = SPSYRK_ERR_HIP;
        } else if (out && mk.phase >= 0 && mk.phase < SPSYRK_NUM_PHASES) {
            out->ms[mk.phase] += ms;
            out->launches[mk.phase] += 1;
        }
        pool_event(mk.a);
        pool_event(mk.b);
    }
    g_marks.clear();
    return st;
}

}  // extern "C"
