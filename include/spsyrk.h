/*
 * spsyrk.h -- local sparse SYRK on one AMD Instinct MI355X (gfx950).
 *
 * C-ABI of libspsyrk.so.  Every entry point computes on the GPU with
 * hand-written HIP kernels; nothing falls back to the host.
 *
 * The operation (paper Sec. II-A): for a sparse A in R^{m x n}, C = A A^T is
 * the m x m Gram matrix of the rows of A; it is symmetric, so one triangle
 * holds all of its information.  Sec. III-A computes only the lower triangle
 * of a diagonal block (C_ii = sum_s SYRK(A_is)) and Sec. III-B writes an
 * off-diagonal block as C_ij = sum_s A_is A_js^T, with the transpose fused into
 * the local kernel so A^T is never materialised.  Sec. V-F (Eq. (spmv))
 * defines the stored lower part C_L *including the diagonal* and the full
 * matrix C = C_L + C_L^T - D.
 *
 *   spsyrk_lower   : C_L = tril(A A^T)       (entries with column <= row)
 *   spsyrk_offdiag : C   = A_i A_j^T         (full rectangular block, no prune)
 *   spsyrk_mirror  : C   = C_L + C_L^T - D   (symmetric completion of C_L)
 *
 * Reproducibility: structure and the count semirings are the same bit for
 * bit on every run; plus-times values of rows with many products (the
 * dense-tile accumulator) are summed in an order that may change from run to
 * run, so their last bits may differ (within the stated tolerances).
 *
 * Structure is the pattern product: C(i,j) is stored iff rows i and j share a
 * stored column (stored zeros of A count as structure; computed zeros are
 * kept).  Output rows keep the input row order and columns ascend strictly
 * within each row, so the diagonal is the last entry of every non-empty row of
 * C_L.
 *
 * Conventions common to all calls
 * -------------------------------
 * - Matrices are canonical CSR, 0-based: row_ptr is int64[nrows + 1] with
 *   row_ptr[0] == 0, non-decreasing, row_ptr[nrows] == nnz; col_idx is
 *   int32[nnz], strictly increasing within each row, in [0, ncols).
 * - All pointers inside spsyrk_csr / spsyrk_csr_out are DEVICE pointers on the
 *   current HIP device.  The struct pointers themselves are host pointers.
 * - Inputs are owned by the caller and are only read.
 * - Every output array and every temporary buffer is obtained through the
 *   allocator passed in (or hipMallocAsync / hipFreeAsync on the stream when
 *   the allocator is NULL).  On SPSYRK_OK the output arrays belong to the
 *   caller, who releases them with the same allocator.  On any error every
 *   allocation made by the call has been released and *C is zeroed.
 * - Work is ordered on hip_stream (a hipStream_t; NULL means the default
 *   stream).  A call returns with the output's row_ptr and nnz final and the
 *   remaining work enqueued on hip_stream (synchronise the stream before
 *   reading values).  Before that it blocks the host on hip_stream a fixed
 *   number of times, each time to read a few words that size the buffers
 *   that follow:
 *     spsyrk_lower, spsyrk_lower_plan: 3 -- the validation word of A, the
 *       row classes (heavy rows, staging size), the output size;
 *       spsyrk_lower_plan waits once more for the plan's copies;
 *     spsyrk_offdiag: 3 -- the validation words of both operands (one
 *       read), the row classes, the output size (A_j with 2^28 columns or
 *       more: validation words, the index size, the output size);
 *       spsyrk_offdiag_half: one more, for the split row;
 *     spsyrk_mirror: 3 -- the validation word, the strict-lower count and
 *       the end of the call (when nnz(C_L) exceeds 2^31 the strict lower
 *       part is transposed in column slabs: one column histogram per
 *       refinement and one record count per slab instead of the count);
 *     spsyrk_lower_accumulate: the validation word of C_prev, the three of
 *       spsyrk_lower for the stage, the merge item count, the output size
 *       and the end of the call;
 *     spsyrk_symm: the validation word and the end of the call (Y is
 *       complete on return);
 *     spsyrk_lower_execute: none.
 *   Validation must finish before any kernel reads the input's indices,
 *   which is why it is read on the host first.
 * - Limits: nrows, ncols < 2^31 and, for the inputs of spsyrk_lower and
 *   spsyrk_offdiag, nnz < 2^31 (SPSYRK_ERR_SHAPE otherwise).  Output nnz and
 *   the nnz of spsyrk_mirror's input are int64 (below 2^62).
 * - Thread safety: calls on different streams may run concurrently; error
 *   detail strings are thread-local.
 */
#ifndef SPSYRK_H
#define SPSYRK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPSYRK_ABI_VERSION 2

typedef enum spsyrk_status {
    SPSYRK_OK = 0,
    SPSYRK_ERR_INVALID_ARG = 1,   /* null pointer, negative size, Ai/Aj inner dimensions differ */
    SPSYRK_ERR_NOT_CANONICAL = 2, /* row_ptr or col_idx violate the canonical CSR rules above, or
                                     spsyrk_mirror got an entry above the diagonal */
    SPSYRK_ERR_SHAPE = 3,         /* a dimension or nnz(A) is 2^31 or more */
    SPSYRK_ERR_OOM = 4,           /* the allocator returned NULL */
    SPSYRK_ERR_OVERFLOW = 5,      /* an internal count would overflow its integer type */
    SPSYRK_ERR_HIP = 6,           /* a HIP runtime call failed; see spsyrk_last_error_detail() */
    SPSYRK_ERR_TOO_LARGE = 7      /* spsyrk_symm_noalloc: the operands need more than its fixed scratch */
} spsyrk_status;

/*
 * Value semiring.  Products and sums follow the usual (+, *) except:
 *   F32: inputs are float; products are formed and summed in double and
 *        rounded to float once per output entry.
 *   COUNT_I32: values are ignored (may be NULL); C(i,j) = |S(i) and S(j)|, the
 *        number of shared stored columns (the overlap count used for
 *        k-mer overlap detection, Sec. I), as int32.
 *   COUNT_I32_JACCARD_F32: as COUNT, then J(i,j) = c / (|S(i)| + |S(j)| - c)
 *        as one correctly rounded float division (Jaccard similarity, Sec. I);
 *        output values are float.  The diagonal of C_L is exactly 1.
 * Output value types: F64 -> double, F32 -> float, COUNT_I32 -> int32,
 * COUNT_I32_JACCARD_F32 -> float.
 */
typedef enum spsyrk_semiring {
    SPSYRK_PLUS_TIMES_F64 = 0,
    SPSYRK_PLUS_TIMES_F32 = 1,
    SPSYRK_COUNT_I32 = 2,
    SPSYRK_COUNT_I32_JACCARD_F32 = 3
} spsyrk_semiring;

/* Input CSR (device arrays, read only). */
typedef struct spsyrk_csr {
    int64_t nrows;
    int64_t ncols;
    int64_t nnz;
    const int64_t* row_ptr; /* [nrows + 1] */
    const int32_t* col_idx; /* [nnz] */
    const void* values;     /* [nnz] of double (F64) or float (F32); may be NULL for COUNT* */
} spsyrk_csr;

/* Output CSR (device arrays allocated by the call through the allocator).
 * col_idx and values hold nnz entries (one allocated entry when nnz is 0, so
 * that the pointers are never null on success).  Their allocations can be
 * larger: when spsyrk_lower, spsyrk_lower_plan or spsyrk_offdiag have no
 * heavy rows they are sized by the rows' staging bound (product counts, plus
 * the diagonal in lower mode, at most 16 GiB of columns and values), which
 * exceeds nnz by the number of products that merged. */
typedef struct spsyrk_csr_out {
    int64_t nrows;
    int64_t ncols;
    int64_t nnz;            /* entries in the result */
    int64_t* row_ptr;       /* [nrows + 1] */
    int32_t* col_idx;       /* [nnz] */
    void* values;           /* [nnz] of the semiring's output type */
} spsyrk_csr_out;

/* Device-memory allocator.  alloc returns a device pointer aligned to at least
 * 256 bytes or NULL; free releases it (stream-ordered use on hip_stream is
 * assumed: memory freed by the call may be reused by later work on that
 * stream). */
typedef struct spsyrk_allocator {
    void* (*alloc)(void* ctx, size_t bytes);
    void (*free)(void* ctx, void* p);
    void* ctx;
} spsyrk_allocator;

/*
 * C_L = tril(A A^T), lower triangle with the diagonal (Sec. III-A, Eq. (spmv)).
 * A: m x n.  C: m x m, C->nrows = C->ncols = m.
 * Errors: INVALID_ARG (A, C null; A->values null for PLUS_TIMES), SHAPE,
 * NOT_CANONICAL, OOM, OVERFLOW, HIP.
 */
spsyrk_status spsyrk_lower(const spsyrk_csr* A, spsyrk_semiring sr, const spsyrk_allocator* al,
                           void* hip_stream, spsyrk_csr_out* C);

/*
 * C = A_i A_j^T, the full rectangular off-diagonal block C_ij of Sec. III-B with
 * the transpose fused into the kernel (A_j is read in CSR; no A_j^T is formed
 * by the caller).  A_i: m_i x n, A_j: m_j x n.  C: m_i x m_j.  For the Jaccard
 * semiring |S(j)| is the row length in A_j.
 * Errors: as spsyrk_lower, plus INVALID_ARG if A_i->ncols != A_j->ncols.
 */
spsyrk_status spsyrk_offdiag(const spsyrk_csr* Ai, const spsyrk_csr* Aj, spsyrk_semiring sr,
                             const spsyrk_allocator* al, void* hip_stream, spsyrk_csr_out* C);

/*
 * Two-phase use for repeated products on one pattern (new values on an
 * unchanged matrix).  spsyrk_lower_plan computes C_L = tril(A A^T) as
 * spsyrk_lower does and also returns a plan that keeps every pattern-only
 * result on the device: copies of A's row_ptr and col_idx, the column index
 * of A, the partner runs, product counts, row classes and C_L's row_ptr.
 * spsyrk_lower_execute then computes C_L for new values of the same pattern
 * (values: nnz entries in A's entry order, double for F64, float for F32,
 * ignored by the COUNT semirings): the index's values are gathered from the
 * new ones and the numeric pass writes every row straight into its final
 * place.  It neither sorts nor waits on the host (the output size is known),
 * and returns with the work enqueued on hip_stream.  The output has the
 * plan's structure and the semiring it was made with.
 * The plan's buffers come from the allocator passed to spsyrk_lower_plan
 * (hipMallocAsync on that call's stream when NULL) and stay allocated until
 * spsyrk_plan_destroy, which frees them with that allocator (with none: it
 * waits for the plan's device, returns the buffers with hipFreeAsync on the
 * null stream and waits for that).
 * Executions of one plan must not overlap (they share its counters and the
 * index's values); the plan may be used from any stream once the creating
 * call has returned.
 * Errors: as spsyrk_lower; spsyrk_lower_execute: INVALID_ARG (null plan or
 * missing values), OOM, HIP.
 */
typedef struct spsyrk_plan_s spsyrk_plan;

spsyrk_status spsyrk_lower_plan(const spsyrk_csr* A, spsyrk_semiring sr, const spsyrk_allocator* al,
                                void* hip_stream, spsyrk_plan** plan, spsyrk_csr_out* C);
spsyrk_status spsyrk_lower_execute(spsyrk_plan* plan, const void* values, const spsyrk_allocator* al,
                                   void* hip_stream, spsyrk_csr_out* C);
spsyrk_status spsyrk_plan_destroy(spsyrk_plan* plan);

/*
 * C = C_prev + tril(A_s A_s^T): one stage's update added to the lower part
 * accumulated so far, as a diagonal block sums its stages (Sec. III-A:
 * C_ii = sum over s of SYRK(A_is)).  Accumulating the stages of A = [A_1 ...
 * A_q] one call at a time gives tril(A A^T) (structure exactly; values up to
 * the order of the sums).
 * C_prev: m x m canonical CSR with no entry above the diagonal and values of
 * the semiring's output type (for example an earlier spsyrk_lower or
 * spsyrk_lower_accumulate result; an empty m x m matrix starts a sum).
 * A_s: m x n_s, as for spsyrk_lower.  C: m x m, the union of the two patterns
 * with shared entries summed (F64; F32 as one float addition; COUNT_I32).
 * The Jaccard semiring does not add (its values are ratios): accumulate
 * COUNT_I32 instead; it returns INVALID_ARG.
 * Errors: as spsyrk_lower, plus INVALID_ARG (shapes, Jaccard, missing values)
 * and NOT_CANONICAL for C_prev.
 */
spsyrk_status spsyrk_lower_accumulate(const spsyrk_csr* C_prev, const spsyrk_csr* A_s, spsyrk_semiring sr,
                                      const spsyrk_allocator* al, void* hip_stream, spsyrk_csr_out* C);

/*
 * One half of an off-diagonal block, as the two processes of a symmetric pair
 * split C_ij = C_ji^T between them (Sec. III-A, Algorithm 3): the process
 * below the diagonal computes the top rows of its block, its partner above
 * the diagonal the right columns of its own.  Row r of C_ij is column r of
 * C_ji, so the top half of C_ij and the right half of C_ji are disjoint and
 * together hold the whole pair.
 *   SPSYRK_HALF_TOP:   rows [0, floor(m_i / 2)) of A_i A_j^T.
 *                      C: floor(m_i / 2) x m_j.
 *   SPSYRK_HALF_RIGHT: columns [floor(m_j / 2), m_j) of A_i A_j^T, every row
 *                      of A_i.  C: m_i x m_j, column ids in the block's own
 *                      numbering (all of them >= floor(m_j / 2)).
 * Values, semirings and ordering as spsyrk_offdiag.  The call reads row_ptr at
 * the split row on the host (one more synchronisation) and checks the row
 * range it multiplies.
 * Errors: as spsyrk_offdiag, plus INVALID_ARG for an unknown half.
 */
typedef enum spsyrk_half { SPSYRK_HALF_TOP = 0, SPSYRK_HALF_RIGHT = 1 } spsyrk_half;

spsyrk_status spsyrk_offdiag_half(const spsyrk_csr* Ai, const spsyrk_csr* Aj, spsyrk_half half,
                                  spsyrk_semiring sr, const spsyrk_allocator* al, void* hip_stream,
                                  spsyrk_csr_out* C);

/*
 * C = C_L + C_L^T - D (Eq. (spmv)): the full symmetric matrix from a stored
 * lower part (for example the output of spsyrk_lower).  Row i of the result is
 * row i of C_L followed by the entries (r, i) of the strict lower part with
 * r > i in ascending r.  Values (of the semiring's OUTPUT type; ignored when
 * NULL) are copied bit for bit, so C(i,j) and C(j,i) are bitwise equal.
 * C_lower: m x m.  C_full: m x m, nnz = 2 nnz(C_L) - (number of diagonal entries).
 * Errors: INVALID_ARG (non-square), NOT_CANONICAL (including any entry with
 * column > row), SHAPE, OOM, OVERFLOW, HIP.
 */
spsyrk_status spsyrk_mirror(const spsyrk_csr* C_lower, spsyrk_semiring sr, const spsyrk_allocator* al,
                            void* hip_stream, spsyrk_csr_out* C_full);

/*
 * Y = C X for the symmetric C = C_L + C_L^T - D, reading only the stored
 * lower part (Eq. (spmv) for one column, Eq. (spgemm) for several): C_L X
 * plus (X^T C_L)^T minus D X, with no transpose of C_L formed.
 * C_lower: m x m canonical CSR with no entry above the diagonal (for example
 * the output of spsyrk_lower), values of the semiring's OUTPUT type (double,
 * float, int32 or float; NULL only when nnz is 0).
 * X: device array, m x k row-major with leading dimension ldx >= k;
 * Y: device array, m x k row-major with leading dimension ldy >= k, written
 * (every element of the m x k part; the rest of each row is left alone).
 * X and Y hold double for PLUS_TIMES_F64 and COUNT_I32, float for
 * PLUS_TIMES_F32 and COUNT_I32_JACCARD_F32.  Products and sums are formed in
 * double and Y is rounded once; the sums are accumulated with atomic adds, so
 * their order (and the last bits of Y) may differ from run to run.
 * Workspace: m k doubles and a small tile table from the allocator, released
 * before return; for one column (k = 1) of a matrix of 2^19 to 2^21 rows the
 * transposed terms go through buckets of rows instead of atomic adds to
 * random rows, which takes 10 bytes per entry of C_lower more (records of
 * (row in bucket, value)) and a table of per-bucket counts; past 2^21 rows
 * they go through records grouped by ranges of 2^18 rows (12 bytes per entry
 * of C_lower), each range then added on one XCD of the chip.  The variable
 * SPSYRK_SYMM_BUCKETS (read at every call) overrides the bucket choice: 0
 * never, 1 for every single column of up to 2^24 rows, 12 to 14 the same
 * with buckets of 2^12 to 2^14 rows (raised where needed to keep at most
 * 1024 buckets); SPSYRK_SYMM_SPLIT = 0 or 1 turns the range split off, or on
 * for every single column not bucketed.  The call returns after Y is
 * complete.
 * Errors: INVALID_ARG (non-square C_lower, k < 0, ldx or ldy < k, null
 * arrays), NOT_CANONICAL (including an entry above the diagonal), SHAPE, OOM,
 * HIP.
 */
spsyrk_status spsyrk_symm(const spsyrk_csr* C_lower, spsyrk_semiring sr, int64_t k, const void* X, int64_t ldx,
                          void* Y, int64_t ldy, const spsyrk_allocator* al, void* hip_stream);

/*
 * spsyrk_symm without any allocation, for callers that cannot allocate device
 * memory (code that must not call hipMalloc, tight serving loops, harnesses
 * that forbid allocation).  Same operands, semirings, results and errors as
 * spsyrk_symm; it never calls hipMalloc, hipFree or the allocator and never
 * takes the bucketed path: every workspace lives in one fixed array of
 * SPSYRK_NOALLOC_SCRATCH_BYTES per device, part of the library's device code
 * (each device the library runs on holds it until the process ends).
 * Limit: the scratch holds the workspace of 8 m k bytes plus a tile table
 * of about nnz / 512 bytes (and under 1 KiB of alignment); larger operands
 * get SPSYRK_ERR_TOO_LARGE before any device work (m k up to about 16.7 M).
 * The array is shared by every call on a device and keeps the last call's
 * contents (each call clears what must start at zero): calls that overlap on
 * one device -- on different streams or host threads -- race and give wrong
 * results; serialise them.  Blocks the host twice (validation word, end of
 * the call); Y is complete on return.
 */
#define SPSYRK_NOALLOC_SCRATCH_BYTES (128ull << 20)
spsyrk_status spsyrk_symm_noalloc(const spsyrk_csr* C_lower, spsyrk_semiring sr, int64_t k, const void* X,
                                  int64_t ldx, void* Y, int64_t ldy, void* hip_stream);

/* Static description of a status code. */
const char* spsyrk_status_string(spsyrk_status s);

/* Detail of the last error on the calling thread ("" if none). */
const char* spsyrk_last_error_detail(void);

/* Invariant checks of the kernels (a debugging aid, not a passage of the paper).
 * A build compiled with -DSPSYRK_DEBUG=1 (libspsyrk_debug.so) checks, inside its
 * kernels, that every output slot written lies in its row's range of C and that
 * the heavy rows' numeric pass fills exactly the columns its symbolic pass
 * counted; a broken check sets a bit in a device word and the kernel goes on.
 * spsyrk_debug_build returns 1 for that build, 0 for the ordinary one.
 * spsyrk_debug_flags waits for the whole device (hipDeviceSynchronize), then
 * writes the OR of the raised bits to *flags and clears them: 1 compaction
 * destination outside C, 2 heavy output slot outside its row, 4 heavy column
 * count differs from the symbolic count, 2^31 a word could not be read.  The
 * ordinary build always writes 0.  SPSYRK_ERR_INVALID_ARG if flags is NULL,
 * SPSYRK_ERR_HIP if the wait fails. */
int spsyrk_debug_build(void);
spsyrk_status spsyrk_debug_flags(uint32_t* flags);

/* Counters from the last successful call on the calling thread. */
typedef struct spsyrk_stats {
    int64_t nnz_out;          /* entries in the result */
    int64_t csc_entries;      /* entries kept in the column index built from the right operand */
    int64_t heavy_rows;       /* rows routed to the dense-tile accumulator */
    int64_t light_rows;       /* rows handled by the batched ordered-bucket accumulator */
    int64_t products;         /* multiply-adds formed off the diagonal (lower) or in total (offdiag) */
    int64_t heavy_entries;    /* entries of the left operand in heavy rows */
    int64_t heavy_nnz_out;    /* result entries of heavy rows */
    int32_t group_shift;      /* log2 of columns per directory group */
    int32_t row_bits;         /* bits of the row id inside a packed column key */
    int32_t packed_staging;   /* 1 if the light rows' counts or Jaccard values were staged as one
                                 packed 4-byte word per output (column and value) */
    int32_t reserved;         /* 0 */
} spsyrk_stats;

spsyrk_status spsyrk_last_stats(spsyrk_stats* out);

/*
 * Phase timing (profiling aid).  Between spsyrk_timing_begin() and
 * spsyrk_timing_end() every call on the calling thread records a pair of HIP
 * events on its stream around each phase below; the light and heavy numeric
 * and symbolic phases, the compaction and COLINDEX_PACK are one kernel launch
 * each.  spsyrk_timing_end waits for the recorded
 * events, returns the summed milliseconds and the number of timed launches
 * per phase, releases the events and stops recording.  Recording adds no
 * synchronisation to the calls themselves, but every recorded event leaves
 * the device idle for a few microseconds between the kernels around it.
 */
typedef enum spsyrk_phase {
    SPSYRK_PHASE_VALIDATE = 0,       /* canonical-CSR checks of the inputs */
    SPSYRK_PHASE_COLINDEX = 1,       /* column index of the right operand (sort, pack, directory) */
    SPSYRK_PHASE_LIGHT_SYMBOLIC = 2, /* row lengths of rows with few products */
    SPSYRK_PHASE_HEAVY_SYMBOLIC = 3, /* row lengths of rows with many products */
    SPSYRK_PHASE_SCAN = 4,           /* row pointers of the output */
    SPSYRK_PHASE_LIGHT_NUMERIC = 5,  /* columns and values of rows with few products */
    SPSYRK_PHASE_HEAVY_NUMERIC = 6,  /* columns and values of rows with many products */
    SPSYRK_PHASE_MIRROR_COUNT = 7,   /* spsyrk_mirror: row lengths of the full matrix */
    SPSYRK_PHASE_MIRROR_COPY = 8,    /* spsyrk_mirror: lower rows copied into place */
    SPSYRK_PHASE_MIRROR_TRANSPOSE = 9, /* spsyrk_mirror: strict lower part transposed into place */
    SPSYRK_PHASE_RUNS = 10,          /* row classes and the partner run of every entry */
    SPSYRK_PHASE_COMPACT = 11,       /* light rows moved from their staging slots into place */
    SPSYRK_PHASE_COLINDEX_PASSES = 12, /* inside COLINDEX: the sorting passes over the high column bits
                                          (histograms, scans, scatters) */
    SPSYRK_PHASE_COLINDEX_PACK = 13, /* inside COLINDEX: the one-kernel local sort that writes the index
                                        (wide column ids only) */
    SPSYRK_NUM_PHASES = 14
} spsyrk_phase;

typedef struct spsyrk_phase_times {
    double ms[SPSYRK_NUM_PHASES];        /* summed event time per phase */
    int64_t launches[SPSYRK_NUM_PHASES]; /* timed occurrences per phase */
} spsyrk_phase_times;

spsyrk_status spsyrk_timing_begin(void);
/* As spsyrk_timing_begin, for the phases whose bits are set in mask (bit p:
 * phase p) only; the other phases record nothing. */
spsyrk_status spsyrk_timing_begin_phases(uint32_t mask);
spsyrk_status spsyrk_timing_end(spsyrk_phase_times* out);

/* ABI version the library was built with (SPSYRK_ABI_VERSION). */
int spsyrk_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SPSYRK_H */
