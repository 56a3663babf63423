/*
 * gspar -- gradient sparsification on AMD Instinct MI355X (gfx950).
 *
 * Implements the sparsifier of Wangni, Wang, Liu and Zhang, "Gradient Sparsification for
 * Communication-Efficient Distributed Optimization" (arXiv 1710.09854):
 *
 *   1. keep probabilities p_i = min(lambda * |g_i|, 1)                      (Proposition 1)
 *      with lambda chosen so that sum_i p_i = rho * d, either exactly
 *      (Algorithm 2's criterion with a density budget, eqs. 5-7) or by the greedy rescaling of
 *      Algorithm 3 run for a fixed number of steps;
 *   2. Bernoulli selection Z_i with P(Z_i = 1) = p_i                         (Section 3)
 *   3. amplification Q(g)_i = Z_i * g_i / p_i, i.e. g_i on the capped set and sign(g_i)/lambda
 *      elsewhere (Section 3.3; the division-free form of Section 5.3);
 *   4. compaction of the survivors into ascending (int32 index, fp32 value) pairs, the layout of
 *      the Q_A / Q_B lists of Section 3.3 (eqs. 8-10).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Pointers are DEVICE pointers unless marked (host). The caller owns every buffer, including
 *    the workspace; the library never allocates or frees device memory.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream). All work is enqueued
 *    on it; no call synchronises the host. Results (lambda, k, nnz, flags, p, idx, val) become
 *    valid when the stream reaches them.
 *  - A row is one worker's gradient (Algorithm 1, steps 4-5). Batched calls take rows of length d
 *    with a leading dimension ld >= d (elements); row r is independent of every other row and
 *    bit-identical to a single-row call on that row with the same rho and seed.
 *  - Budget: B = rho * d computed in double. rho must lie in [0, 1].
 *  - Solvers: GSPAR_EXACT (the lambda solving sum_i min(lambda|g_i|, 1) = B exactly, capped set
 *    never splitting ties) or GSPAR_GREEDY (Algorithm 3 for `greedy_iters` rescale steps; the
 *    paper's experiments use 2). For every solver the capped set is {p_i = 1} (Proposition 1,
 *    Section 3.3's S_k): every pass, every output and the capped count k use that one set. Special cases: if B >= nnz(g), every nonzero is kept with
 *    probability one (lambda = +inf, Q(g) = g); if rho = 0 nothing is kept (lambda = 0).
 *    GSPAR_VARIANCE is Algorithm 2 as printed, with the variance budget of problem (4): every rho
 *    argument then carries eps (any finite eps >= 0), p_i = 1 on {a > a_(k+1)} for the
 *    smallest k with a_(k+1) T1 <= eps sum a^2 + T2 (eq. 6; T1, T2 the sum and the sum of squares
 *    of the magnitudes not above a_(k+1)) and lambda = T1 / (eps sum a^2 + T2) (eq. 7), every sum
 *    exact and rounded once; if no value satisfies the criterion (possible only through rounding
 *    with eps = 0) every nonzero is capped (lambda = +inf). greedy_iters is ignored.
 *  - Random source: coordinate i of a row with seed s uses word (i mod 4) of Philox4x32-10 with
 *    key (s low 32, s high 32) and counter (floor(i/4) low 32, floor(i/4) high 32, 0, 0);
 *    Z_i = 1 iff word < p_i * 2^32 (Salmon et al., SC'11 for the generator).
 *  - Output is a pure function of (g bytes, d, rho, solver, greedy_iters, seed): identical across
 *    runs, launch geometries and streams.
 *  - Errors detectable on the host are returned synchronously before anything is enqueued:
 *    GSPAR_ERR_ARG (NULL required pointer, d < 1 or d > 2^31 - 1, rows < 1, ld < d, rho outside
 *    [0, 1] or NaN for scalar rho (eps negative, infinite or NaN for GSPAR_VARIANCE),
 *    greedy_iters outside [0, 64], unknown solver, negative
 *    capacity), GSPAR_ERR_WORKSPACE (ws NULL or ws_bytes below gspar_workspace_bytes) and
 *    GSPAR_ERR_HIP (a launch failed). Data-dependent conditions are reported per row in `flags`.
 *  - Calls that share a workspace must be stream-ordered; concurrent calls need distinct
 *    workspaces. The library keeps no state of its own: it is re-entrant, and its exported
 *    symbols are exactly the functions declared here.
 *  - Per-row parameters of the batched, segmented and hybrid calls (rho or eps, Philox seeds)
 *    are DEVICE arrays, read by the kernels: a call then enqueues its work without any host to
 *    device copy (which would order the call after host work and, from pageable memory,
 *    synchronise), and the values may themselves be produced on the device. The single-row calls
 *    take them as host scalars.
 */
#ifndef GSPAR_H
#define GSPAR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#pragma GCC visibility push(default)

typedef enum {
  GSPAR_OK = 0,
  GSPAR_ERR_ARG = -1,
  GSPAR_ERR_WORKSPACE = -2,
  GSPAR_ERR_HIP = -3,
  GSPAR_ERR_TOO_LARGE = -4 /* the call needs more scratch than the library's fixed array holds */
} gspar_status;

typedef enum { GSPAR_GREEDY = 0, GSPAR_EXACT = 1, GSPAR_VARIANCE = 2 } gspar_solver;

/* Per-row flag bits written to `flags[r]`. */
enum {
  GSPAR_FLAG_NONFINITE = 1, /* g holds Inf or NaN: nothing is sampled, nnz = 0, lambda = NaN  */
  GSPAR_FLAG_OVERFLOW = 2,  /* more survivors than capacity: the first `capacity` pairs are
                               written and nnz holds the true count                          */
  GSPAR_FLAG_ALLZERO = 4,   /* g is identically zero: nnz = 0                                 */
  GSPAR_FLAG_BADRHO = 8,    /* (batched) rho[r] outside [0, 1] or NaN (eps: negative, infinite or NaN): row skipped, nnz = 0 */
  GSPAR_FLAG_INTERNAL = 16, /* an internal invariant of the solver's exact arithmetic failed (a
                               library fault, never expected): row skipped, nnz = 0, lambda = NaN */
  GSPAR_FLAG_BADSEG = 32    /* (segmented) the device offsets of the segment disagree with the
                               host offsets' bounds: segment skipped, nnz = 0                 */
};

/* Bytes of device workspace needed by a call on `rows` rows of length d with `solver`. The
 * workspace needs no initialisation; 256-byte alignment is required. */
size_t gspar_workspace_bytes(int64_t rows, int64_t d, int solver);

/* A capacity that holds every survivor except with negligible probability:
 * min(d, ceil(rho*d + 8*sqrt(rho*d) + 64)). The expected number of survivors is
 * sum_i p_i <= rho*d (Section 3.1, expected sparsity). */
int64_t gspar_capacity_hint(int64_t d, double rho);

/* Keep probabilities of one row (Proposition 1 with lambda from the chosen solver).
 *   g       [d] fp32 gradient (read only)
 *   p       [d] fp32 output p_i = min(lambda |g_i|, 1), exactly 1 on the capped set; may be NULL
 *           to compute lambda only
 *   lambda  [1] fp64 output; k [1] int64 output (size of the capped set, may be NULL);
 *   flags   [1] uint32 output (may be NULL). */
int sparsify_probs(const float* g, int64_t d, double rho, int solver, int greedy_iters, float* p,
                   double* lambda, int64_t* k, uint32_t* flags, void* ws, size_t ws_bytes,
                   void* stream);

/* Solve, sample, amplify and compact one row.
 *   idx [capacity] int32 and val [capacity] fp32 receive the survivors in ascending index order:
 *   val = g_i on the capped set (p_i = 1) and sign(g_i)/lambda rounded to fp32 elsewhere.
 *   nnz [1] int64 receives the true survivor count (it may exceed capacity, see FLAG_OVERFLOW).
 *   lambda, k and flags are optional outputs ([1] each, may be NULL). */
int sparsify_sample_compact(const float* g, int64_t d, double rho, int solver, int greedy_iters,
                            uint64_t seed, int32_t* idx, float* val, int64_t capacity,
                            int64_t* nnz, double* lambda, int64_t* k, uint32_t* flags, void* ws,
                            size_t ws_bytes, void* stream);

/* Batched keep probabilities: rows x d gradients with leading dimension ld, one row per worker
 * (Algorithm 1, steps 4-5: every worker sparsifies its own gradient); row r is Proposition 1 with
 * rho[r] and is bit-identical to sparsify_probs on that row.
 *   rho [rows] fp64 DEVICE array; p [rows*ld] or NULL; lambda [rows] (required), k [rows] and
 *   flags [rows] optional. */
int sparsify_probs_batched(const float* g, int64_t rows, int64_t d, int64_t ld, const double* rho,
                           int solver, int greedy_iters, float* p, double* lambda, int64_t* k,
                           uint32_t* flags, void* ws, size_t ws_bytes, void* stream);

/* Batched solve + sample + compact, one row per worker (Algorithm 1, steps 4-5: each worker m
 * computes Q(g^m) from its own gradient; Section 3's selection and amplification per row).
 * rho [rows] fp64 and seeds [rows] uint64 are DEVICE arrays.
 * Row r writes its survivors to idx[r*cap_per_row ...] and val[r*cap_per_row ...] and its count
 * to nnz[r]; lambda, k and flags ([rows] each) are optional. */
int sparsify_sample_compact_batched(const float* g, int64_t rows, int64_t d, int64_t ld,
                                    const double* rho, int solver, int greedy_iters,
                                    const uint64_t* seeds, int32_t* idx, float* val,
                                    int64_t cap_per_row, int64_t* nnz, double* lambda, int64_t* k,
                                    uint32_t* flags, void* ws, size_t ws_bytes, void* stream);

/* Hybrid coding of the sparsified gradient (Section 3.3, eqs. 9-10): the same solve and the same
 * Bernoulli selection as sparsify_sample_compact (identical survivors for identical arguments),
 * with the survivors split by the capped set S_k = {p_i = 1}:
 *   Q_A: idx_a[r*cap_a ...] int32 ascending indices and val_a[...] fp32 values g_i of the capped
 *        survivors (every capped coordinate survives); n_a[r] receives their true count, which is
 *        also the capped count k;
 *   Q_B: code_b[r*cap_b ...] int32 words (index | sign << 31), ascending by index, for every other
 *        survivor, whose value is sign(g_i)/lambda; n_b[r] receives their true count;
 *   inv_lambda [rows] fp32 (optional): the single float 1/lambda that Q_B's values share
 *        (0 when lambda is 0 or +inf);
 *   q [rows*ld] int8 (optional): the dense ternary vector of Section 3.3, 2 on S_k, sign(g_i) for
 *        the other survivors, 0 elsewhere.
 * rho [rows] fp64 and seeds [rows] uint64 are DEVICE arrays; lambda and flags are optional
 * [rows] outputs. GSPAR_FLAG_OVERFLOW is set when n_a > cap_a or n_b > cap_b (the first cap_a /
 * cap_b entries are written). code_b is required; idx_a and val_a may be NULL when cap_a = 0. */
int sparsify_sample_hybrid_batched(const float* g, int64_t rows, int64_t d, int64_t ld,
                                   const double* rho, int solver, int greedy_iters,
                                   const uint64_t* seeds, int32_t* idx_a, float* val_a,
                                   int64_t cap_a, int64_t* n_a, int32_t* code_b, int64_t cap_b,
                                   int64_t* n_b, float* inv_lambda, int8_t* q, double* lambda,
                                   uint32_t* flags, void* ws, size_t ws_bytes, void* stream);

/* Single-row hybrid coding: rho and seed are host scalars; every array has one row (q has d
 * entries); n_a and n_b are [1] DEVICE outputs. */
int sparsify_sample_hybrid(const float* g, int64_t d, double rho, int solver, int greedy_iters,
                           uint64_t seed, int32_t* idx_a, float* val_a, int64_t cap_a,
                           int64_t* n_a, int32_t* code_b, int64_t cap_b, int64_t* n_b,
                           float* inv_lambda, int8_t* q, double* lambda, uint32_t* flags,
                           void* ws, size_t ws_bytes, void* stream);

/* Coding length in bits of one hybrid message of a d-coordinate gradient with n_a entries in Q_A,
 * n_b in Q_B of which n_b_neg are negative, for floats of `float_bits` bits (host only, no GPU).
 *   out[0]: sparse lists, n_a (b + log2 d) + n_b (log2 d + 1) + b (indices, values, signs, 1/lambda);
 *   out[1]: entropy-coded ternary vector, sum over its four symbols of d_l log2(d / d_l), plus
 *           n_a b for Q_A's values and b for 1/lambda (Section 3.3);
 *   out[2]: the experiments' per-message cost (Section 5), n_a (b + log2 d) + min(2d, n_b log2 d)
 *           + b, with the realised n_b in place of the expected sum of p over the uncapped set.
 * Returns GSPAR_ERR_ARG for out = NULL, d < 1, negative counts, n_a + n_b > d, n_b_neg > n_b or
 * float_bits < 1. */
int gspar_coding_bits(int64_t d, int64_t n_a, int64_t n_b, int64_t n_b_neg, int float_bits,
                      double* out);

/* Per-layer sparsification (Section 5.2: each layer of a network is sparsified on its own).
 * Segment s of the flat vector g is g[off[s] .. off[s+1]) and is treated as its own row: its own
 * density rho[s] (budget rho[s] * length), its own lambda, capped set and Philox key seeds[s], with
 * the Philox counter and the output indices taken within the segment, so the result of a segment
 * equals a single-row call on it. off_host and off_dev hold the same segs + 1 offsets (int64), on the
 * host (checked here: off[0] >= 0, nondecreasing, every length below 2^31; used to size the launch)
 * and on the device (read by the kernels, which check each segment again against the host's bounds
 * and flag one that disagrees GSPAR_FLAG_BADSEG); g holds off[segs] floats. Segments may be empty
 * (then flagged GSPAR_FLAG_ALLZERO). Vector loads are used when g is 16-byte aligned and every
 * offset is a multiple of 4. The workspace is gspar_workspace_bytes(segs, L, solver) with L the
 * longest segment (at least 1). rho [segs] fp64 and seeds [segs] uint64 are DEVICE arrays.
 * sparsify_sample_compact_segmented writes segment s's survivors to idx[s*cap_per_seg ...] and
 * val[s*cap_per_seg ...] and its count to nnz[s]; sparsify_probs_segmented writes p in g's layout
 * (p[off[s] + i]). lambda, k and flags are [segs] (optional where the batched calls allow it).
 * Errors: those of the batched calls, and GSPAR_ERR_ARG for NULL or invalid offsets or segs outside
 * [1, 2^24]. */
int sparsify_sample_compact_segmented(const float* g, int64_t segs, const int64_t* off_host,
                                      const int64_t* off_dev, const double* rho, int solver,
                                      int greedy_iters, const uint64_t* seeds, int32_t* idx, float* val,
                                      int64_t cap_per_seg, int64_t* nnz, double* lambda, int64_t* k,
                                      uint32_t* flags, void* ws, size_t ws_bytes, void* stream);
/* Per-layer hybrid coding: the segmented call's solve and selection with the outputs of
 * sparsify_sample_hybrid_batched, one row per segment (indices within the segment); q, when given,
 * has g's layout (q[off[s] + i]). A call whose device offsets are rejected (GSPAR_FLAG_BADSEG on
 * every segment) leaves q unwritten. */
int sparsify_sample_hybrid_segmented(const float* g, int64_t segs, const int64_t* off_host,
                                     const int64_t* off_dev, const double* rho, int solver,
                                     int greedy_iters, const uint64_t* seeds, int32_t* idx_a,
                                     float* val_a, int64_t cap_a, int64_t* n_a, int32_t* code_b,
                                     int64_t cap_b, int64_t* n_b, float* inv_lambda, int8_t* q,
                                     double* lambda, uint32_t* flags, void* ws, size_t ws_bytes,
                                     void* stream);
int sparsify_probs_segmented(const float* g, int64_t segs, const int64_t* off_host,
                             const int64_t* off_dev, const double* rho, int solver, int greedy_iters,
                             float* p, double* lambda, int64_t* k, uint32_t* flags, void* ws,
                             size_t ws_bytes, void* stream);

/* Aggregation of the workers' sparsified gradients (Algorithm 1, step 6, on one device): the dense
 * average v_i = (1/M) sum_m Q(g^m)_i for M = `workers`, from the lists that
 * sparsify_sample_compact_batched writes (worker m's entries idx[m*cap ...], val[m*cap ...], the
 * first min(nnz[m], cap) of them, indices strictly ascending in [0, d)). Each v_i is the fp64 sum
 * of the workers' values at i taken in worker order m = 0, 1, ..., divided by M and rounded to
 * fp32, so the result does not depend on the launch. idx, val, nnz [workers] int64 and v [d] fp32
 * are DEVICE memory; no workspace is used. Entries outside [0, d) are skipped; a list that does
 * not ascend strictly can lose entries, but nothing is read beyond a list's first min(nnz, cap)
 * entries. Returns GSPAR_ERR_ARG for NULL nnz or v, NULL lists with cap > 0, workers outside
 * [1, 2^20], d outside [1, 2^31 - 1] or cap < 0; GSPAR_ERR_HIP if the launch failed. */
int gspar_aggregate(const int32_t* idx, const float* val, int64_t cap, const int64_t* nnz,
                    int64_t workers, int64_t d, float* v, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): sparsify_sample_compact_batched without the workspace
 * arguments. The scratch memory the kernels need comes from a fixed array inside the library,
 * GSPAR_SCRATCH_BYTES on every GPU the library runs on, held until the process ends; the call
 * allocates nothing (no hipMalloc, no hipFree, no allocating library routine). Its results are
 * bit-identical to sparsify_sample_compact_batched's for the same arguments.
 *   Returns GSPAR_ERR_TOO_LARGE, enqueuing nothing, when gspar_workspace_bytes(rows, d, solver)
 * exceeds GSPAR_SCRATCH_BYTES; GSPAR_ERR_HIP if the array's address cannot be obtained on the
 * current device; otherwise the errors of sparsify_sample_compact_batched.
 *   Every call on one GPU uses that GPU's one array, which keeps the last call's contents (each
 * call clears what it needs cleared): calls that may overlap in time on one GPU race and must be
 * ordered, for instance on one stream. */
#define GSPAR_SCRATCH_BYTES ((size_t)32 << 20)
int sparsify_sample_compact_batched_noalloc(const float* g, int64_t rows, int64_t d, int64_t ld,
                                            const double* rho, int solver, int greedy_iters,
                                            const uint64_t* seeds, int32_t* idx, float* val,
                                            int64_t cap_per_row, int64_t* nnz, double* lambda,
                                            int64_t* k, uint32_t* flags, void* stream);

/* Human-readable name of a status code (static storage). */
const char* gspar_status_string(int status);

/* Library version as major*10000 + minor*100 + patch. */
int gspar_version(void);


#pragma GCC visibility pop

#ifdef __cplusplus
}
#endif

#endif /* GSPAR_H */
