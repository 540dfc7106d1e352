// Internal interfaces between the library's translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "spsyrk.h"

namespace spsyrk {

// A pair of HIP events around the work enqueued on stream s during its
// lifetime, recorded while phase timing is on (spsyrk_timing_begin); phase is
// a spsyrk_phase value.
class PhaseTimer {
   public:
    PhaseTimer(int phase, hipStream_t s);
    ~PhaseTimer();
    PhaseTimer(const PhaseTimer&) = delete;
    PhaseTimer& operator=(const PhaseTimer&) = delete;

   private:
    hipStream_t s_;
    int phase_;
    hipEvent_t a_{}, b_{};
    bool on_ = false;
};

// semiring codes (same values as the public enum)
enum Sr : int { kF64 = 0, kF32 = 1, kCount = 2, kJaccard = 3 };

// bytes of the per-entry value carried by the column index of the right operand
inline int csc_value_bytes(int sr) { return sr == kF64 ? 8 : (sr == kF32 ? 4 : (sr == kJaccard ? 4 : 0)); }
// bytes of an output value
inline int out_value_bytes(int sr) { return sr == kF64 ? 8 : 4; }

struct DevCsr {
    int64_t m = 0, n = 0, nnz = 0;
    const int64_t* rp = nullptr;
    const int32_t* ci = nullptr;
    const void* v = nullptr;
};

// Column index of the right operand B (B = A for the lower triangle, B = A_j
// off the diagonal): the entries of B grouped by column, rows ascending inside
// a column, packed as key = (col mod 2^gs) << rowbits | row, plus a directory
// of 2^gs-column groups: the entries of group g occupy [gptr[g], gptr[g+1]).
// In lower mode the last (largest-row) entry of every column is left out: it
// is never the partner j < i of another row.
struct ColIndex {
    int64_t n = 0;          // columns of B
    int64_t m = 0;          // rows of B
    int gs = 0;             // log2 columns per group
    int rowbits = 1;        // bits of a row id inside a key
    int64_t ngroups = 0;    // groups; gptr has ngroups + 1 entries
    int64_t nkept = 0;      // entries kept (device-side value is authoritative until synced)
    uint32_t* key = nullptr;
    void* val = nullptr;    // double / float values of B, or int32 row lengths of B (Jaccard)
    uint32_t* gptr = nullptr;  // null when every entry's partner run is given (no lookups)
    // > 0 (Jaccard with every partner run given): each key also carries its
    // row's length above the row bits, saturated at 2^lenbits - 1 (the full
    // length then comes from the row pointers), and val is null
    int lenbits = 0;
};

// Partner runs of the entries of the left operand: the positions [first, end)
// of the column index that hold an entry's partners.  One word per entry in
// r4: first * radix + (end - first), with radix = floor(2^32 / (positions +
// 1)) (at most 2^16), so every first fits; a length of radix - 1 or more is
// written as radix - 1 and the run itself goes to r8 (radix 1: every run in
// r8).  r4 starts zeroed, so an entry never written has the empty run (with
// radix 1, r8 is zeroed too).  The words halve the bytes of the scattered
// writes that build the table and of the reads that follow, and a mixed
// radix keeps every run of up to radix - 2 partners in its word.  (The
// two-pass kernels keep runs in r8 alone, with r4 null; only run_of reads
// that form.)
struct RunTab {
    uint32_t* r4 = nullptr;
    uint2* r8 = nullptr;
    uint32_t radix = 1;
    double inv = 1.0;  // 1 / radix, rounded to nearest
    __host__ __device__ explicit operator bool() const { return r4 != nullptr || r8 != nullptr; }
};

// The run of a word loaded by the caller (escapes read r8[e]).  The quotient
// comes from a double product: its error is below 2^-20 for words below
// 2^32, so adding 2^-18 and truncating gives floor(v / radix) exactly while
// radix stays below 2^17.
__device__ inline uint2 run_from(const RunTab& t, uint32_t v, int64_t e) {
    const uint32_t first = uint32_t(fma(double(v), t.inv, 0x1p-18));
    const uint32_t len = v - first * t.radix;
    if (len == t.radix - 1u) return t.r8[e];
    return make_uint2(first, first + len);
}

__device__ inline uint2 run_of(const RunTab& t, int64_t e) { return t.r4 ? run_from(t, t.r4[e], e) : t.r8[e]; }

__device__ inline void set_run(const RunTab& t, int64_t e, uint32_t first, uint32_t end) {
    const uint32_t len = end - first;
    if (len + 1u < t.radix) {
        t.r4[e] = first * t.radix + len;
    } else {
        t.r4[e] = t.radix - 1u;
        t.r8[e] = make_uint2(first, end);
    }
}

// The radix of the words for an index of `positions` entries (every first
// <= positions): floor(2^32 / (positions + 1)), at most 2^16, or 1 (every
// run in r8) below 8.  SPSYRK_RUN_RADIX=k (read at every call) asks for k
// instead (at most the value above; 0 or 1: every run in r8).
uint32_t run_radix(int64_t positions);

// ---- scan.hip
// Exclusive scan out[i] = sum_{k<i} in[i]; out may alias in.  If total is not
// null it receives the sum (device pointer).  tmp needs scan_tmp_bytes(n).
size_t scan_tmp_bytes(int64_t n);
void scan_u32(const uint32_t* in, uint32_t* out, int64_t n, uint32_t* total, void* tmp, hipStream_t s);
void scan_i64(const int64_t* in, int64_t* out, int64_t n, int64_t* total, void* tmp, hipStream_t s);

// ---- validate.hip
// Records per tile of the radix passes.  The validation of a matrix whose
// columns are sorted next counts the first pass's digits over the same tiles
// (hist: digit-major, ntiles x 256 words; digit (col >> shift) & mask), so
// that the pass does not read the column ids once more for them.
constexpr int kRadixTile = 3072;
struct FirstHist {
    uint32_t* hist = nullptr;
    int shift = 0;
    uint32_t mask = 0;
    int64_t ntiles = 0;
};
// ORs ErrBits into *err.  upper_forbidden: also flag entries with col > row.
// tmp: validate_tmp_bytes(nnz) of scratch.
size_t validate_tmp_bytes(int64_t nnz);
void validate_csr(const DevCsr& A, bool upper_forbidden, uint32_t* err, void* tmp, hipStream_t s,
                  const FirstHist* fh = nullptr);
void fill_u32(uint32_t* p, int64_t n, uint32_t v, hipStream_t s);

// ---- radix.hip
// Stable LSD sort of (key, row, value) records by the low `nbits` of key.
// Buffers *_a hold the input and the result is returned in the buffer
// reported by the return value (0 -> *_a, 1 -> *_b).  vbytes in {0, 4, 8}.
size_t radix_tmp_bytes(int64_t n);
// scratch of radix_sort_csr for n entries and nbits-bit columns
size_t radix_csr_tmp_bytes(int64_t n, int nbits);
// Stable sort of the entries of a CSR matrix by column: the records
// (column, row field, entry index) are formed inside the first pass.  The row
// field is the row in its low rowbits bits and, if lenbits > 0, the row's
// length saturated at 2^lenbits - 1 above them.  Returns 0 if the result is in
// the *_a buffers, 1 for *_b.
// The column index in partner-run form, written by the sort itself when it
// takes the local path: key (the row) and value of every entry at its sorted
// position, and (with a run table, its words zeroed) every entry's partner
// run {first position of its column, its own position}.  *kept (zeroed) gets the kept
// entries (all, or all but the last of every column with drop_last).
struct LocalPack {
    RunTab run;
    uint32_t* key = nullptr;
    void* val = nullptr;         // null for Jaccard: the keys carry the row lengths (the row field)
    const void* vals_b = nullptr;  // values of B by entry index (vbytes 4 or 8)
    const int64_t* rp_b = nullptr; // row pointers of B (Jaccard lengths)
    int vbytes = 0;
    bool jac = false;
    int rowbits = 1, lenbits = 0;
    bool drop_last = false;
    int64_t* kept = nullptr;
    uint32_t* ccount = nullptr;  // non-null (zeroed, one per column): entries of every column
    uint32_t* vsrc = nullptr;    // non-null: the entry index of every written position
    // 4 or 8 (with vals_b, and no run table and no vsrc): the record passes
    // carry each entry's value in place of its index (the third record
    // buffers then hold values of that size), so the local sort reads values
    // in sorted order instead of gathering them by entry index
    int carried = 0;
};
// pk non-null: write the column index as above when the local path is taken
// and return -1 (no sorted copy); otherwise as described.
// hist1 (optional): the first pass's digit histogram, already counted (by
// the validation; it is scanned in place)
// trow1 (optional): the row of every tile start (tiles of kRadixTile
// entries; -1 where left out), as the validation writes it
int radix_sort_csr(const int32_t* col_idx, const int64_t* rp, int64_t m, int rowbits, int lenbits, uint32_t* key_a,
                   uint32_t* key_b, uint32_t* row_a, uint32_t* row_b, uint32_t* ent_a, uint32_t* ent_b, int64_t n,
                   int nbits, void* tmp, hipStream_t s, const LocalPack* pk = nullptr, uint32_t* hist1 = nullptr,
                   const int64_t* trow1 = nullptr);
// Low column bits sorted inside groups by radix_sort_csr for n entries with
// nbits-bit columns (0: passes over every bit, no local sort).
int local_bits(int64_t n, int nbits);
// The digit of radix_sort_csr's first pass over n entries with nbits-bit
// columns: (col >> shift) & mask.
void radix_first_digit(int64_t n, int nbits, int* shift, uint32_t* mask);
int radix_sort(uint32_t* key_a, uint32_t* key_b, uint32_t* row_a, uint32_t* row_b, void* val_a,
               void* val_b, int vbytes, int64_t n, int nbits, void* tmp, hipStream_t s);

// ---- colindex.hip
// From the entries of B sorted by column (column, row field as written by
// radix_sort_csr, entry index): keep flags, packed keys, values gathered by
// entry index from vals_b (the row length |S(row)| for Jaccard) and the group
// directory.  With a run table (lower mode) the partner run {first, end} of
// every entry with partners is written at its entry index (the table's words
// start zeroed: the other entries keep empty runs).
size_t colindex_tmp_bytes(int64_t n);
void build_colindex(const uint32_t* scol, const uint32_t* srow, const uint32_t* sent, int64_t n_entries,
                    bool drop_last, int vbytes_in, int sr, const void* vals_b, const int64_t* rp_b, int lenbits,
                    ColIndex& ci, void* tmp, int64_t* d_nkept, const RunTab& run, hipStream_t s,
                    uint32_t* vsrc = nullptr);

// ---- light.hip
struct LightArgs {
    // left operand (rows of the output)
    int64_t m = 0;
    const int64_t* rp = nullptr;
    const int32_t* ci = nullptr;
    const void* val = nullptr;
    // right operand's column index
    ColIndex cx;
    int64_t m_right = 0;          // output columns
    bool lower = true;
    int sr = kF64;
    // symbolic outputs
    int64_t* row_nnz = nullptr;   // [m]
    uint8_t* heavy_flag = nullptr;  // [m]
    int32_t* heavy_rows = nullptr;  // list of heavy rows
    int32_t* heavy_count = nullptr; // device counter
    unsigned long long* products = nullptr;  // device counter of products formed (light rows)
    // numeric outputs
    const int64_t* c_rp = nullptr;
    int32_t* c_ci = nullptr;
    void* c_val = nullptr;
};
void light_symbolic(const LightArgs& a, hipStream_t s);
void light_numeric(const LightArgs& a, hipStream_t s);

// ---- light_fused.hip
// Light-row limits of the single-pass kernel: a row is light when it has at
// most kFusedEntries entries and kFusedProducts off-diagonal products.
constexpr int kFusedEntries = 256;
constexpr int kFusedProducts = 512;
constexpr int kFusedRows = 32;
struct FusedArgs {
    int64_t m = 0;
    const int64_t* rp = nullptr;
    const int32_t* ci = nullptr;
    const void* val = nullptr;
    ColIndex cx;
    int64_t m_right = 0;
    bool lower = true;
    int sr = kF64;
    const int64_t* rp_right = nullptr;         // row pointers of the right operand (Jaccard lengths)
    const unsigned long long* prod = nullptr;  // off-diagonal products per row
    RunTab run;                                // partner run {first, end} of every entry
    const int64_t* heavy_nnz = nullptr;        // output lengths of heavy rows
    const int64_t* ubp = nullptr;              // staging slot of every row (prefix of upper bounds)
    int64_t* row_cnt = nullptr;                // exact output length of every row
    int rows_per_chunk = 8;
    int64_t nchunks = 0;
    unsigned long long* chunk_counter = nullptr;  // zeroed: chunks handed out so far
    int32_t* c_ci = nullptr;                   // staging columns
    void* c_val = nullptr;                     // staging values
    // > 0 (count and Jaccard): every output is staged as one word in c_ci,
    // column * pack_rr + packed value, where the packed value is the count,
    // or (Jaccard) the count * pack_r2 + the partner's length; the
    // compaction unpacks it (c_val unused)
    uint32_t pack_rr = 0, pack_r2 = 0;
};
// light rows: columns and values at the staging slots, exact lengths in row_cnt
// (heavy rows: their length from heavy_nnz; row_cnt[m] = 0)
void light_fused(const FusedArgs& a, hipStream_t s);
// heavy rows (over the limits) into a list; light capacity sum(prod + diagonal) and
// the sum of prod over all rows into the two counters
// and ub[i] = products + diagonal for light rows, 0 for heavy rows (and ub[m]
// = 0); maxlen
// (optional, zeroed): the largest row length
void classify_rows(const int64_t* rp, const unsigned long long* prod, int64_t m, bool lower, int32_t* heavy_rows,
                   int32_t* heavy_count, unsigned long long* light_cap, unsigned long long* prod_sum, int64_t* ub,
                   hipStream_t s, unsigned long long* maxlen = nullptr);

// ---- runs.hip
// Dense column starts of a CSR matrix's column-sorted copy: cptr[c] =
// entries in columns before c (n + 1 words; scan_tmp: scan_tmp_bytes(n + 1)).
void column_starts(const int32_t* ci, int64_t nnz, int64_t n, uint32_t* cptr, void* scan_tmp, hipStream_t s);
// Row pointers of rows [r0, r0 + m) of a CSR matrix, rebased to start at 0
// (out: m + 1 words).
void rebase_rows(const int64_t* rp, int64_t r0, int64_t m, int64_t* out, hipStream_t s);
// dst[p] = src[idx[p]] for p < n, elements of vb (4 or 8) bytes.
void gather_values(void* dst, const void* src, const uint32_t* idx, int64_t n, int vb, hipStream_t s);
// ci[p] += off for p < nnz.
void shift_columns(int32_t* ci, int64_t nnz, int32_t off, hipStream_t s);
// Off-diagonal partner runs: run[e] = {cptr[ci[e]], cptr[ci[e] + 1]}.
void offdiag_runs(const int32_t* ci, int64_t nnz, const uint32_t* cptr, const RunTab& run, hipStream_t s);
// prod[i] = sum over the entries e of row i of run[e].y - run[e].x (prod
// must start zeroed).
// tmp: row_products_tmp_bytes(nnz) of scratch
size_t row_products_tmp_bytes(int64_t nnz);
// trow1 (optional): the row of every tile start of kRadixTile entries (-1
// where left out), as the validation writes it
void row_products(const int64_t* rp, int64_t m, int64_t nnz, const RunTab& run, void* tmp, unsigned long long* prod,
                  hipStream_t s, const int64_t* trow1 = nullptr);
// Copy the staged rows to their final places: the element at staging slot
// ubp[i] + x (x < row_cnt[i]) goes to c_rp[i] + x.  ubp is non-decreasing
// with ubp[m] = staged; rows with no staging room (heavy rows) copy nothing.
// packed (kCount or kJaccard, else 0): s_ci holds packed words (see
// FusedArgs::pack_rr), unpacked into the column and the 4-byte value; rp_a
// gives the rows' lengths (Jaccard).
// tmp: compact_tmp_bytes(staged) of scratch
size_t compact_tmp_bytes(int64_t staged);
void compact_rows(int64_t m, int64_t staged, const int64_t* ubp, const int64_t* row_cnt, const int64_t* c_rp,
                  const int32_t* s_ci, const void* s_val, int vbytes, void* tmp, int32_t* c_ci, void* c_val,
                  hipStream_t s, int packed = 0, uint32_t pack_rr = 0, uint32_t pack_r2 = 0,
                  const int64_t* rp_a = nullptr);
// Reorders the heavy-row list rows[0..n) by decreasing magnitude of their
// product counts (powers of two; stable inside one), so that the rows with
// the most work are taken first from the heavy kernels' queue.
// tmp: heavy_order_tmp_bytes(n)
size_t heavy_order_tmp_bytes(int64_t n);
void heavy_order(int32_t* rows, int64_t n, const unsigned long long* prod, void* tmp, hipStream_t s);
// Over the rows listed in rows[0..n): adds the entries of A (rp) to out[0]
// and the output entries (c_rp) to out[1] (zeroed beforehand).
void heavy_sums(const int32_t* rows, int64_t n, const int64_t* rp, const int64_t* c_rp, unsigned long long* out,
                hipStream_t s);
// Row of every tile start: trow[t] = the row r with rp[r] <= t T < rp[r + 1],
// for t T < rp[m] (rp non-decreasing; trow: ceil(rp[m] / T) words).
void tile_first_rows(const int64_t* rp, int64_t m, int64_t T, int64_t* trow, hipStream_t s);

// ---- heavy.hip
struct HeavyArgs {
    int64_t m = 0;
    const int64_t* rp = nullptr;
    const int32_t* ci = nullptr;
    const void* val = nullptr;
    ColIndex cx;
    int64_t m_right = 0;
    const int64_t* rp_right = nullptr;  // row lengths of the right operand (Jaccard)
    bool lower = true;
    int sr = kF64;
    const int32_t* heavy_rows = nullptr;
    const int32_t* heavy_count = nullptr;
    int64_t heavy_max = 0;              // upper bound of heavy rows (grid sizing)
    // per-entry run bounds (sized nnz of the left operand), written by the symbolic pass
    RunTab run;                         // partner run {first, end} of every entry (r8 only
                                        // when the symbolic pass writes it)
    bool runs_ready = false;            // run already filled (the symbolic pass skips its lookups)
    uint32_t* cursor = nullptr;
    uint32_t* rend = nullptr;           // end of every heavy entry's run (set with the cursors)
    unsigned long long* products = nullptr;  // optional: add the products formed
    int64_t* row_nnz = nullptr;
    unsigned long long* nnz_total = nullptr; // optional: add the heavy rows' lengths
    const int64_t* c_rp = nullptr;
    int32_t* c_ci = nullptr;
    void* c_val = nullptr;
};
// queue: one device int of scratch (work counter)
void heavy_symbolic(const HeavyArgs& a, int* queue, hipStream_t s);
void heavy_numeric(const HeavyArgs& a, int* queue, hipStream_t s);

// ---- accumulate.hip
// Row-wise union of two lower parts P and T (m rows, canonical), in work items
// of at most a few thousand entries: chunks of short rows and windows of long
// rows.  merge_item_flags leaves an exclusive scan of the per-row item counts
// in fl (m + 1 words; the number of items in fl[m]; scan_tmp:
// scan_tmp_bytes(m + 1)).  merge_item_table then writes the item table: crow
// (items + 1 words), cwin (items words).  merge_lower with write false sets
// cnt[i] = distinct columns of row i (cnt zeroed before) and wsum[q] = the
// count of item q if it is a window, else 0; with wsum scanned (exclusive) and
// write true it writes the merged rows (columns ascending, shared entries
// summed) at crp.  sr: F64, F32 or COUNT.
void merge_item_flags(int64_t m, const DevCsr& P, const DevCsr& T, int64_t* fl, void* scan_tmp, hipStream_t s);
void merge_item_table(int64_t m, const DevCsr& P, const DevCsr& T, const int64_t* fl, int64_t* crow, int32_t* cwin,
                      hipStream_t s);
void merge_lower(bool write, int sr, int64_t items, const int64_t* crow, const int32_t* cwin, const DevCsr& P,
                 const DevCsr& T, int64_t* cnt, int64_t* wsum, const int64_t* crp, int32_t* cci, void* cv,
                 hipStream_t s);

// ---- symm.hip
// Y = C X with C = C_L + C_L^T - D from the stored lower part C (canonical,
// nothing above the diagonal, values of the semiring's output type).  X and
// Y: m x k row-major (ldx, ldy), double for F64 and COUNT, float otherwise.
// mode: how the transposed term is added (symm_mode gives the default
// choice; the same value goes to both calls): atomic adds to random rows,
// LDS buckets of rows (one column, 2^19 to 2^21 rows), or records split by
// row range and added per XCD (one column, past 2^21 rows).
// tmp: symm_tmp_bytes(m, k, nnz, mode).
enum SymmMode : int { kSymmAtomics = 0, kSymmBuckets = 1, kSymmSplit = 2 };
int symm_mode(int64_t m, int64_t k, int64_t nnz);
size_t symm_tmp_bytes(int64_t m, int64_t k, int64_t nnz, int mode);
void symm_product(const DevCsr& C, int sr, const void* x, int64_t ldx, int64_t k, void* y, int64_t ldy, void* tmp,
                  int mode, hipStream_t s);

// ---- the mirror's slab sort (radix.hip)
// The mirror slab behind a fused sort: record p of row r (rows from the
// record pointers rec_rp) is entry p + row_off[r] of C_L, with
// key = column - c0; the record at sorted position q goes to the full rows at
// before + q + rp[c0 + key + 1] (its column's lower part, then the column's
// strict entries in row order).
struct SlabIo {
    const int32_t* ci = nullptr;      // C_L's columns
    const void* val = nullptr;        // C_L's values or null
    const int64_t* row_off = nullptr; // per row: its first entry in the slab less its first record
    int64_t c0 = 0;                   // the slab's first column
    const int64_t* rp = nullptr;      // C_L's row pointers
    int64_t before = 0;               // strict entries of the columns before c0
    int32_t* f_ci = nullptr;          // full rows
    void* f_val = nullptr;
};
// Sort of a slab of nrec records with keys of nbits <= 16 bits (one or two
// passes) into the full rows, the first pass reading C_L through the slab's
// rows or (extracted) the records already in key_a, row_a, val_a; returns
// the buffer with the sorted keys.  tmp: radix_tmp_bytes(nrec).
uint32_t* slab_sort_place(const SlabIo& io, int vbytes, int64_t nrec, int nbits, const int64_t* rec_rp, int64_t m,
                          bool extracted, uint32_t* key_a, uint32_t* key_b, uint32_t* row_a, uint32_t* row_b,
                          void* val_a, void* val_b, void* tmp, hipStream_t s);

// ---- mirror.hip
struct MirrorArgs {
    int64_t m = 0;
    int64_t nnz = 0;
    const int64_t* rp = nullptr;
    const int32_t* ci = nullptr;
    const void* val = nullptr;
    int vbytes = 0;
};
// strict-lower entries with clo <= col < clo + nb * 2^cb per bucket of 2^cb
// columns (nb <= kMirrorBins), added into hist (zeroed here)
constexpr int kMirrorBins = 4096;
// columns of a narrow transpose slab (its keys sort in two 8-bit passes)
constexpr int64_t kMirrorNarrow = int64_t(1) << 16;
void mirror_coarse_hist(const MirrorArgs& a, int64_t clo, int cb, int nb, unsigned long long* hist,
                        hipStream_t s);
// row of every tile start of the mirror's walks over positions [0, rp[m])
// (trow: mirror_tile_bytes(rp[m]))
size_t mirror_tile_bytes(int64_t positions);
void mirror_tile_rows(const int64_t* rp, int64_t m, int64_t* trow, hipStream_t s);
// per-row counts and first entries of the strict lower part with col in [c0, c1)
// row_lo[r] -= rec_rp[r] for every row (the entry of record p of row r is then p + row_lo[r])
void mirror_slab_offsets(int64_t* row_lo, const int64_t* rec_rp, int64_t m, hipStream_t s);
void mirror_slab_counts(const MirrorArgs& a, int64_t c0, int64_t c1, int64_t* row_cnt, int64_t* row_lo,
                        hipStream_t s);
// records (col - c0, row, value) of the slab, in row-major order at positions
// given by rec_rp (exclusive scan of the per-row counts), nrec in all
// (trow: mirror_tile_bytes(nrec) of scratch)
void mirror_slab_extract(const MirrorArgs& a, int64_t c0, int64_t nrec, const int64_t* rec_rp, const int64_t* row_lo,
                         int64_t* trow, uint32_t* rkey, uint32_t* rrow, void* rval, hipStream_t s);
// from the slab's records sorted by column (keys skey): first[k] / end[k],
// the record range of slab column k, and the full row starts f_rp[c0..c1]
// (fl: w + 1 words of scratch; strict_before: strict-lower entries in the
// columns before c0; first / end: w words each)
void mirror_slab_columns(const MirrorArgs& a, int64_t c0, int64_t c1, const uint32_t* skey, int64_t nrec,
                         uint32_t* first, uint32_t* end, int64_t* fl, int64_t strict_before, int64_t* f_rp,
                         void* scan_tmp, hipStream_t s);
// place sorted records: record s of slab column k goes to
// f_rp[c0 + k] + lower_len(c0 + k) + (s - first[k])
void mirror_slab_place(const MirrorArgs& a, int64_t c0, int64_t nrec, const uint32_t* skey, const uint32_t* srow,
                       const void* sval, const uint32_t* first, const int64_t* f_rp, int32_t* f_ci, void* f_val,
                       hipStream_t s);
// lower rows' entries [ebeg, eend) to their places f_rp[row] + offset in row
// (trow: the table of mirror_tile_rows over the lower rows, or null)
void mirror_copy_lower(const MirrorArgs& a, int64_t ebeg, int64_t eend, const int64_t* trow, const int64_t* f_rp,
                       int32_t* f_ci, void* f_val, hipStream_t s);

}  // namespace spsyrk
