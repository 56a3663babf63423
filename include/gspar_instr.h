/*
 * gspar measurement build -- libgspar_instr.so, the same source as libgspar.so compiled with
 * GSPAR_INSTRUMENT. It exports every function of gspar.h unchanged, plus the hooks below. They
 * are for the benchmark and the tests only: they keep process-global state (not thread-safe) and
 * are therefore absent from the product library, whose exports are exactly gspar.h.
 */
#ifndef GSPAR_INSTR_H
#define GSPAR_INSTR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#pragma GCC visibility push(default)

/* Kernel classes reported by gspar_prof_read, in this order (GSPAR_PROF_CLASSES of them):
 * 0 sampling / compaction, 1 statistics pass, 2 probabilities, 3 solver, 4 refinement pass,
 * 5 workspace initialisation, 6 aggregation, 7 per-row outputs of the probabilities calls,
 * 8 row sample for the candidate band. */
#define GSPAR_PROF_CLASSES 9

/* Arms the launch timer: each of the next `max_launches` kernel launches (any entry point, any
 * stream) is made with hipExtLaunchKernelGGL and a pair of HIP events that the dispatch itself
 * stamps at the kernel's start and end. Returns GSPAR_ERR_ARG for max_launches < 1 and
 * GSPAR_ERR_HIP if the events cannot be created. */
int gspar_prof_arm(int max_launches);
/* Waits for the last armed launch and writes, per class, the summed kernel time in ms
 * (ms[GSPAR_PROF_CLASSES]) and the number of launches (launches[GSPAR_PROF_CLASSES]). */
int gspar_prof_read(double* ms, int* launches);
/* Releases the events; later launches are untimed. */
int gspar_prof_disarm(void);

/* Host-compiled copies of the device arithmetic, for CPU tests:
 * the 320-bit accumulator rounded to double (limbs5: 5 little-endian 64-bit limbs, unit 2^-149); */
double gspar_check_fx_round(const uint64_t* limbs5);
/* v * 2^s into limbs5; returns 16 (the internal-invariant flag) and zero limbs for s outside
 * [0, 255]; */
uint32_t gspar_check_fx_shifted(uint64_t v, int s, uint64_t* limbs5);
/* (qh * 2^24 + ql) * 2^(2 shift) into limbs10 (unit 2^-298); 16 and zero limbs for 2 shift
 * outside [0, 511]; */
uint32_t gspar_check_fq_squares(uint64_t qh, uint64_t ql, int shift, uint64_t* limbs10);
/* the exact sum of |x_i| over the finite nonzero entries, rounded once to double; */
double gspar_check_exact_sum(const float* x, int64_t n);
/* the smallest key t with fl(lambda * value(t)) >= 1 (0x7F800000 when none); */
uint32_t gspar_check_cap_key(double lam);
/* Philox4x32-10 of counter ctr[4] under key[2]. */
void gspar_check_philox(const uint32_t* ctr, const uint32_t* key, uint32_t* out);

/* Stream probe on `stream` (not timed here; the caller brackets it with events): with dst NULL,
 * reads the n floats of src (device, 16-byte aligned, n a multiple of 4) and adds their sum to
 * *sink (device double); otherwise copies them to dst (device, 16-byte aligned, not overlapping
 * src). A plain kernel that reads (or reads and writes) each byte once, to compare the path's
 * bandwidth with. Returns GSPAR_ERR_ARG for bad pointers or sizes. */
int gspar_probe_stream(const float* src, float* dst, int64_t n, double* sink, void* stream);

#pragma GCC visibility pop

#ifdef __cplusplus
}
#endif

#endif /* GSPAR_INSTR_H */
