/*
 * phsa_prof.h - the profiling build of libphsa.
 *
 * libphsa_prof.so holds the same kernels and the same C ABI as libphsa.so
 * (include/phsa.h) and, in addition, the calls below.  While recording is on,
 * every kernel launch is bracketed by a pair of HIP events on the stream it is
 * launched on, so a caller can read each kernel's own duration.  It is a
 * measurement tool for benchmarks; the product library, libphsa.so, exports
 * none of this and keeps no state.
 *
 * Unlike libphsa.so this build keeps process-wide state (the recorded events),
 * guarded by a mutex; phsa_prof_durations synchronises the events it reads.
 * Kernel names are the profiling names of the launchers ("phsa_select",
 * "phsa_attn_bwd_sparse", ...).
 */
#ifndef PHSA_PROF_H
#define PHSA_PROF_H

#include <stdint.h>

#include "phsa.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Starts (enable != 0) or stops recording launches.  Event objects are
 * created as needed and reused after phsa_prof_reset. */
PHSA_API phsa_status phsa_prof_enable(int32_t enable);

/* Waits for the recorded launches of kernel `name` and writes the duration of
 * each, in milliseconds and in launch order, to ms[0 .. min(n, cap) - 1];
 * returns n, the number of launches recorded for `name` (ms may be NULL when
 * cap is 0). */
PHSA_API int32_t phsa_prof_durations(const char *name, float *ms, int32_t cap);

/* Drops every record (events go back to a pool). */
PHSA_API void phsa_prof_reset(void);

#ifdef __cplusplus
}
#endif

#endif /* PHSA_PROF_H */
