/*
 * fpo_prof.h - opt-in kernel timing of libfpo (measurement instrumentation;
 * not an operation of the method).
 *
 * When enabled, every library kernel whose name matches the filter is
 * bracketed by two hipEvents recorded on the stream it is launched on, so the
 * interval is that kernel's execution on the device. fpo_prof_read waits for
 * the recorded events and reports the accumulated milliseconds and launch
 * count per kernel name. Disabled (the default) the launch path does nothing
 * extra. The registry is process-wide and guarded by a mutex.
 *
 * Kernel names: rms_forward, logits_chunk, chunk_stats, proj_chunk,
 * finalize_vjp, transpose_pad, outer, errh, reduce_parts, update,
 * update_reduce, cosine, cosine_reduce.
 */
#ifndef FPO_PROF_H
#define FPO_PROF_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* filter: NULL or "" times every kernel; otherwise a comma-separated list of
 * kernel names. Returns 0. */
int fpo_prof_enable(const char* filter);
/* Stop timing new launches (already recorded events stay readable). */
int fpo_prof_disable(void);
/* Wait for all recorded events, fold them into the per-name totals and copy
 * up to max_entries of them out: names[i] (NUL-terminated, 32 bytes each),
 * total_ms[i], launches[i]. Returns the number of names with data, or a
 * negative value if a HIP event call failed. Totals persist until reset. */
int fpo_prof_read(int max_entries, char* names, double* total_ms, int64_t* launches);
/* Drop all totals and pending events. */
int fpo_prof_reset(void);

#ifdef __cplusplus
}
#endif

#endif /* FPO_PROF_H */
